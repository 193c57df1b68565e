"""Packed byte format, version 1, written out plainly (test infrastructure only).

The paper stores each group's codes as packed low-bit bytes, never expanded to
fp16 in memory (section 6, "Fused kernels over packed weights" and
"Granularity is deployment-friendly"), but leaves the byte format open.  This
module restates the format this repository fixes, independently of the C++
packer, so that the two can be compared byte for byte:

  G = K/64 group columns; class c = log2(b) (0:1-bit .. 3:8-bit).
  R = tile rows (power of two), T = ceil(N/R) row tiles.
  C = groups per column chunk, U = ceil(G/C) chunks.
  Unit u = t*U + k covers rows [tR, min(N,tR+R)) and group columns
  [kC, min(G,kC+C)); inside it, position p = (j-kC)*R + (r-tR).
  Codes are offset-binary: u = q + 2^(b-1) (b >= 2), u = (q+1)/2 (b = 1).

  Sections, in this order, each at a 256-byte aligned offset; every byte not
  written below is zero; the blob length is rounded up to 256:
    0 unit table  uint32[n_units+1][8]  {e0,e1,e2,e3, wmap_word, 0,0,0}
    1 wmap        uint64 words; per unit W_u = ceil(C_k*R/64) words of plane 0
                  (class bit 0) then W_u words of plane 1 (class bit 1);
                  position p is bit p%64 of word p/64
    2..5 codes[c] entries of class c ordered by (unit, p); entry = 2b uint32
                  little-endian words; pair i (weights 2i, 2i+1) in word
                  i // (16/b), field f = i % (16/b): weight 2i in bits
                  [f*b, f*b+b), weight 2i+1 in bits [16+f*b, 16+f*b+b)
    6..9 scales[c] fp16 bit patterns (uint16) in the same entry order
"""

import numpy as np

from .quant import G, WIDTHS, offset_code, level_from_code

ALIGN = 256
N_SECTIONS = 10


def _ceil_div(a, b):
    return -(-a // b)


def _align(n):
    return _ceil_div(n, ALIGN) * ALIGN


def geometry(N, K, tile_rows, chunk_groups):
    """Tile / chunk / unit counts of the format."""
    Gc = K // G
    T = _ceil_div(N, tile_rows)
    U = _ceil_div(Gc, chunk_groups)
    return {"N": N, "K": K, "G": Gc, "R": tile_rows, "C": chunk_groups,
            "T": T, "U": U, "units": T * U}


def _unit_positions(geo, t, k):
    """Yield (p, r, j) for every real (non-padding) position of unit (t, k), in p order."""
    R, C = geo["R"], geo["C"]
    j0, j1 = k * C, min(geo["G"], (k + 1) * C)
    for j in range(j0, j1):
        for rl in range(R):
            r = t * R + rl
            if r < geo["N"]:
                yield (j - j0) * R + rl, r, j


def _unit_words(geo, k):
    C = geo["C"]
    Ck = min(geo["G"], (k + 1) * C) - k * C
    return _ceil_div(Ck * geo["R"], 64)


def encode_record(u, b):
    """Pack the 64 offset codes of one group into its 2b uint32 words."""
    per_word = 16 // b
    words = [0] * (2 * b)
    for i in range(32):
        wi, f = divmod(i, per_word)
        words[wi] |= int(u[2 * i]) << (f * b)
        words[wi] |= int(u[2 * i + 1]) << (16 + f * b)
    return words


def decode_record(words, b):
    """Inverse of encode_record: the 64 offset codes of one group."""
    per_word = 16 // b
    mask = (1 << b) - 1
    u = [0] * 64
    for i in range(32):
        wi, f = divmod(i, per_word)
        u[2 * i] = (int(words[wi]) >> (f * b)) & mask
        u[2 * i + 1] = (int(words[wi]) >> (16 + f * b)) & mask
    return u


def _encode_records(U, b):
    """Vectorised encode_record over entries: U int64[E, 64] -> uint32[E, 2b]."""
    per_word = 16 // b
    E = U.shape[0]
    words = np.zeros((E, 2 * b), dtype=np.uint64)
    for i in range(32):
        wi, f = divmod(i, per_word)
        words[:, wi] |= U[:, 2 * i].astype(np.uint64) << np.uint64(f * b)
        words[:, wi] |= U[:, 2 * i + 1].astype(np.uint64) << np.uint64(16 + f * b)
    return words.astype(np.uint32)


def pack(q, s_bits, bits, tile_rows, chunk_groups):
    """Pack levels q int[N][K], fp16 scales s_bits uint16[N][K/64] and the bit map.

    Returns (blob uint8[], info dict) where info holds the geometry, per-class
    entry counts, section offsets / lengths and the total length.
    """
    q = np.asarray(q, dtype=np.int64)
    s_bits = np.asarray(s_bits, dtype=np.uint16)
    bits = np.asarray(bits, dtype=np.int64)
    N, K = q.shape
    geo = geometry(N, K, tile_rows, chunk_groups)
    cls_of = {1: 0, 2: 1, 4: 2, 8: 3}

    entries = [[] for _ in range(4)]  # (r, j) per class in (unit, p) order
    unit_rows = []
    wmap_words = []
    for t in range(geo["T"]):
        for k in range(geo["U"]):
            unit_rows.append([len(entries[0]), len(entries[1]), len(entries[2]),
                              len(entries[3]), len(wmap_words), 0, 0, 0])
            W = _unit_words(geo, k)
            plane0 = [0] * W
            plane1 = [0] * W
            for p, r, j in _unit_positions(geo, t, k):
                c = cls_of[int(bits[r, j])]
                if c & 1:
                    plane0[p // 64] |= 1 << (p % 64)
                if c & 2:
                    plane1[p // 64] |= 1 << (p % 64)
                entries[c].append((r, j))
            wmap_words.extend(plane0)
            wmap_words.extend(plane1)
    unit_rows.append([len(entries[0]), len(entries[1]), len(entries[2]),
                      len(entries[3]), len(wmap_words), 0, 0, 0])

    sections = [np.array(unit_rows, dtype=np.uint32).tobytes(),
                np.array(wmap_words, dtype=np.uint64).tobytes()]
    codes, scales = [], []
    for c, b in enumerate(WIDTHS):
        if entries[c]:
            rows = np.array([e[0] for e in entries[c]])
            cols = np.array([e[1] for e in entries[c]])
            qg = q.reshape(N, K // G, G)[rows, cols]  # [E, 64]
            Ug = (qg + 1) // 2 if b == 1 else qg + (1 << (b - 1))
            codes.append(_encode_records(Ug, b).tobytes())
            scales.append(s_bits[rows, cols].astype(np.uint16).tobytes())
        else:
            codes.append(b"")
            scales.append(b"")
    sections += codes + scales

    offs, lens, pos = [], [], 0
    for sec in sections:
        pos = _align(pos)
        offs.append(pos)
        lens.append(len(sec))
        pos += len(sec)
    total = _align(pos)
    blob = np.zeros(total, dtype=np.uint8)
    for off, sec in zip(offs, sections):
        blob[off:off + len(sec)] = np.frombuffer(sec, dtype=np.uint8)
    info = dict(geo)
    info.update({"n_entries": [len(e) for e in entries], "section_off": offs,
                 "section_len": lens, "total_bytes": total})
    return blob, info


def unpack(blob, info):
    """Recover (q int8[N][K], s_bits uint16[N][K/64], bits uint8[N][K/64]) from a blob.

    Walks the unit table and the width map position by position; the codes
    are read with decode_record.  Raises ValueError on any inconsistency.
    """
    blob = np.asarray(blob, dtype=np.uint8)
    N, K = info["N"], info["K"]
    geo = geometry(N, K, info["R"], info["C"])
    off, ln = info["section_off"], info["section_len"]
    units = np.frombuffer(blob[off[0]:off[0] + ln[0]].tobytes(), dtype=np.uint32).reshape(-1, 8)
    wmap = np.frombuffer(blob[off[1]:off[1] + ln[1]].tobytes(), dtype=np.uint64)
    code_words = [np.frombuffer(blob[off[2 + c]:off[2 + c] + ln[2 + c]].tobytes(), dtype=np.uint32)
                  for c in range(4)]
    scale_arr = [np.frombuffer(blob[off[6 + c]:off[6 + c] + ln[6 + c]].tobytes(), dtype=np.uint16)
                 for c in range(4)]
    q = np.zeros((N, K), dtype=np.int8)
    s = np.zeros((N, K // G), dtype=np.uint16)
    bits = np.zeros((N, K // G), dtype=np.uint8)
    for t in range(geo["T"]):
        for k in range(geo["U"]):
            u = t * geo["U"] + k
            nxt = [int(units[u, c]) for c in range(4)]
            w0 = int(units[u, 4])
            W = _unit_words(geo, k)
            for p, r, j in _unit_positions(geo, t, k):
                b0 = (int(wmap[w0 + p // 64]) >> (p % 64)) & 1
                b1 = (int(wmap[w0 + W + p // 64]) >> (p % 64)) & 1
                c = b0 | (b1 << 1)
                b = WIDTHS[c]
                e = nxt[c]
                nxt[c] += 1
                words = code_words[c][e * 2 * b:(e + 1) * 2 * b]
                us = decode_record(words, b)
                q[r, j * G:(j + 1) * G] = [level_from_code(v, b) for v in us]
                s[r, j] = scale_arr[c][e]
                bits[r, j] = b
            for c in range(4):
                if nxt[c] != int(units[u + 1, c]):
                    raise ValueError("unit table inconsistent with the width map")
    return q, s, bits


def code_bytes(bits):
    """Bytes of the code sections: 8*b per group (sum over the bit map)."""
    return int(np.sum(8 * np.asarray(bits, dtype=np.int64)))


def offset_codes(q, b):
    """Offset codes of a whole group (list) at width b."""
    return [offset_code(int(v), b) for v in q]
