// Geometry of the packed layout (version 1, declared in include/vbq.h), shared
// by the host packer and the device launchers of libvbq.
#pragma once

#include <cstdint>
#include "../../include/vbq.h"

namespace vbq {

constexpr int kGroup = 64;
constexpr int kAlign = 256;          // section alignment in bytes
constexpr int kMaxChunk = 128;       // max group columns per unit
constexpr int kMaxUnitPositions = 8192;  // R * C bound (LDS budget of one unit)
constexpr int kUnitRowWords = 8;     // uint32 per unit-table row

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline uint64_t align_up(uint64_t n) { return (n + kAlign - 1) / kAlign * kAlign; }
inline bool is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

struct Geometry {
  int64_t N = 0, K = 0, G = 0;   // rows, columns, group columns
  int32_t R = 0, C = 0;          // tile rows, chunk groups
  int64_t T = 0, U = 0, units = 0;
  int64_t wmap_words = 0;        // total 64-bit words of the width map

  // group columns of chunk k
  int64_t chunk_cols(int64_t k) const {
    int64_t j0 = k * C, j1 = j0 + C < G ? j0 + C : G;
    return j1 - j0;
  }
  // 64-bit words per plane of a unit in chunk k
  int64_t unit_words(int64_t k) const { return ceil_div(chunk_cols(k) * R, 64); }
  int64_t tile_rows(int64_t t) const {
    int64_t r0 = t * R;
    return N - r0 < R ? N - r0 : R;
  }
};

// Library choice of tile rows / chunk groups, and validation of caller choices.
inline vbq_status make_geometry(int64_t N, int64_t K, const vbq_pack_opts* o, Geometry* g) {
  if (N < 1 || K < kGroup || K % kGroup != 0) return VBQ_ERR_SHAPE;
  if (N > (int64_t)1 << 31 || K > (int64_t)1 << 26) return VBQ_ERR_SHAPE;
  g->N = N;
  g->K = K;
  g->G = K / kGroup;
  int32_t R = o ? o->tile_rows : 0;
  int32_t C = o ? o->chunk_groups : 0;
  if (R == 0) {
    // enough row tiles to spread one matrix over the 256 CUs several times;
    // 64-row tiles from 448 of them up (measured on MI355X: a 28672 x 4096
    // matrix runs 8% faster in 448 tiles of 64 rows than in 896 of 32)
    R = 16;
    if (ceil_div(N, 32) >= 512) R = 32;
    if (ceil_div(N, 64) >= 448) R = 64;
  }
  if (!is_pow2(R) || R < 16 || R > 256) return VBQ_ERR_UNSUPPORTED;
  if (C == 0) {
    // one unit per wave of the one-row kernel: at least four units per tile,
    // each at most 32 group columns wide, the count a multiple of four (a
    // unit's entries of each class are one run of the unit table, so a wave
    // that owns a whole unit needs no class counts of its own)
    int64_t U = ceil_div(g->G, 32);
    U = U < 4 ? 4 : (U + 3) / 4 * 4;
    C = (int32_t)ceil_div(g->G, U);
    int64_t cmax = kMaxUnitPositions / R < kMaxChunk ? kMaxUnitPositions / R : kMaxChunk;
    if (C > cmax) C = (int32_t)cmax;
  }
  if (C < 1 || C > kMaxChunk || (int64_t)R * C > kMaxUnitPositions) return VBQ_ERR_UNSUPPORTED;
  g->R = R;
  g->C = C;
  g->T = ceil_div(N, R);
  g->U = ceil_div(g->G, C);
  g->units = g->T * g->U;
  int64_t per_tile = 0;
  for (int64_t k = 0; k < g->U; ++k) per_tile += 2 * g->unit_words(k);
  g->wmap_words = per_tile * g->T;
  return VBQ_OK;
}

inline int class_of_bits(uint8_t b) {
  switch (b) {
    case 1: return 0;
    case 2: return 1;
    case 4: return 2;
    case 8: return 3;
    default: return -1;
  }
}

// Section sizes from the per-class entry counts; fills offsets, lengths, total.
inline void layout_sections(const Geometry& g, const int64_t n_entries[4], vbq_desc* d) {
  uint64_t len[VBQ_NSECTIONS];
  len[VBQ_SEC_UNITS] = (uint64_t)(g.units + 1) * kUnitRowWords * 4;
  len[VBQ_SEC_WMAP] = (uint64_t)g.wmap_words * 8;
  for (int c = 0; c < 4; ++c) {
    len[VBQ_SEC_CODES0 + c] = (uint64_t)n_entries[c] * (8u << c);
    len[VBQ_SEC_SCALES0 + c] = (uint64_t)n_entries[c] * 2;
  }
  uint64_t pos = 0;
  for (int s = 0; s < VBQ_NSECTIONS; ++s) {
    pos = align_up(pos);
    d->section_off[s] = pos;
    d->section_len[s] = len[s];
    pos += len[s];
  }
  d->total_bytes = align_up(pos);
}

inline void fill_desc_header(const Geometry& g, const int64_t n_entries[4], vbq_desc* d) {
  *d = vbq_desc{};
  d->magic = VBQ_MAGIC;
  d->version = VBQ_LAYOUT_VERSION;
  d->N = g.N;
  d->K = g.K;
  d->group = kGroup;
  d->tile_rows = g.R;
  d->chunk_groups = g.C;
  d->n_tiles = g.T;
  d->n_chunks = g.U;
  d->n_units = g.units;
  for (int c = 0; c < 4; ++c) d->n_entries[c] = n_entries[c];
  layout_sections(g, n_entries, d);
}

}  // namespace vbq
