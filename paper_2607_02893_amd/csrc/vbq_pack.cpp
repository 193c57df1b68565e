// Host-side quantizer and packer of libvbq (layout version 1, include/vbq.h).
//
// vbq_pack quantizes each 64-weight group as in paper section 3.1 (Eq. (1) for
// b in {2,4,8}, sign times absmean for b = 1) and writes the packed blob;
// vbq_pack_codes packs levels that were quantized elsewhere.  Both run in two
// passes over row tiles on host threads: count the groups of each width per
// unit, then write every section at its final offset.

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <thread>
#include <vector>

#include "vbq_layout.hpp"

using namespace vbq;

namespace {

struct Counts {
  std::vector<uint32_t> per_unit;  // [units][4]
};

// Run fn(t) for every tile t on up to n_threads host threads.
template <class F>
void parallel_tiles(int64_t T, uint32_t n_threads, F&& fn) {
  unsigned hw = std::thread::hardware_concurrency();
  int64_t nt = n_threads ? n_threads : (hw ? hw : 1);
  nt = std::min<int64_t>(std::min<int64_t>(nt, 64), T);
  if (nt <= 1) {
    for (int64_t t = 0; t < T; ++t) fn(t);
    return;
  }
  std::atomic<int64_t> next{0};
  std::vector<std::thread> pool;
  for (int64_t i = 0; i < nt; ++i)
    pool.emplace_back([&] {
      for (int64_t t; (t = next.fetch_add(1)) < T;) fn(t);
    });
  for (auto& th : pool) th.join();
}

void record_error(std::atomic<int>& err, vbq_status s) {
  int expected = VBQ_OK;
  err.compare_exchange_strong(expected, (int)s);
}

// Count the groups of each class per unit and validate the bit map.
vbq_status count_units(const Geometry& g, const uint8_t* bits, uint32_t n_threads, Counts* out) {
  out->per_unit.assign((size_t)g.units * 4, 0);
  std::atomic<int> err{VBQ_OK};
  parallel_tiles(g.T, n_threads, [&](int64_t t) {
    if (err.load(std::memory_order_relaxed) != VBQ_OK) return;
    int64_t rows = g.tile_rows(t);
    for (int64_t k = 0; k < g.U; ++k) {
      uint32_t* cnt = &out->per_unit[(size_t)(t * g.U + k) * 4];
      int64_t j0 = k * g.C, cols = g.chunk_cols(k);
      for (int64_t rl = 0; rl < rows; ++rl) {
        const uint8_t* brow = bits + (t * g.R + rl) * g.G + j0;
        for (int64_t jl = 0; jl < cols; ++jl) {
          int c = class_of_bits(brow[jl]);
          if (c < 0) {
            record_error(err, VBQ_ERR_BITS);
            return;
          }
          cnt[c]++;
        }
      }
    }
  });
  return (vbq_status)err.load();
}

// Prefix sums of the counts into per-unit starting entries, and the totals.
vbq_status unit_starts(const Geometry& g, const Counts& cnt, std::vector<uint32_t>* starts,
                       int64_t n_entries[4]) {
  starts->assign((size_t)(g.units + 1) * 4, 0);
  uint64_t run[4] = {0, 0, 0, 0};
  for (int64_t u = 0; u <= g.units; ++u) {
    for (int c = 0; c < 4; ++c) {
      if (run[c] > 0xFFFFFFFFull) return VBQ_ERR_UNSUPPORTED;
      (*starts)[(size_t)u * 4 + c] = (uint32_t)run[c];
      if (u < g.units) run[c] += cnt.per_unit[(size_t)u * 4 + c];
    }
  }
  for (int c = 0; c < 4; ++c) n_entries[c] = (int64_t)run[c];
  if ((uint64_t)g.wmap_words > 0xFFFFFFFFull) return VBQ_ERR_UNSUPPORTED;
  return VBQ_OK;
}

// Word offset of unit (t, k) in the width-map section.
int64_t wmap_offset(const Geometry& g, int64_t t, int64_t k) {
  int64_t per_tile = 0, before = 0;
  for (int64_t kk = 0; kk < g.U; ++kk) {
    if (kk == k) before = per_tile;
    per_tile += 2 * g.unit_words(kk);
  }
  return t * per_tile + before;
}

inline uint16_t to_fp16_bits(double v) {
  _Float16 h = (_Float16)v;  // one correctly rounded (nearest-even) conversion
  uint16_t b;
  std::memcpy(&b, &h, 2);
  return b;
}

inline double fp16_to_double(uint16_t b) {
  _Float16 h;
  std::memcpy(&h, &b, 2);
  return (double)h;
}

inline bool fp16_finite(uint16_t b) { return (b & 0x7C00u) != 0x7C00u; }

// Encode 64 offset codes of width b (2b words): pair i -> word i/(16/b),
// field i%(16/b); even weight in the low half-word, odd weight in the high.
inline void encode_record(const uint8_t* u, int b, uint8_t* dst) {
  const int per_word = 16 / b;
  uint32_t words[16];
  for (int w = 0; w < 2 * b; ++w) words[w] = 0;
  for (int i = 0; i < 32; ++i) {
    int wi = i / per_word, f = i % per_word;
    words[wi] |= (uint32_t)u[2 * i] << (f * b);
    words[wi] |= (uint32_t)u[2 * i + 1] << (16 + f * b);
  }
  std::memcpy(dst, words, (size_t)8 * b);
}

// Quantize one group (paper section 3.1).  Writes offset codes u[64] and the
// fp16 scale; returns a status.
inline vbq_status quantize_group(const float* w, int b, uint8_t* u, uint16_t* s_bits) {
  for (int i = 0; i < kGroup; ++i)
    if (!std::isfinite(w[i])) return VBQ_ERR_NONFINITE;
  if (b == 1) {
    double sum = 0.0;
    for (int i = 0; i < kGroup; ++i) sum += std::fabs((double)w[i]);
    uint16_t sb = to_fp16_bits(sum / kGroup);
    if (!fp16_finite(sb)) return VBQ_ERR_SCALE_RANGE;
    *s_bits = sb;
    for (int i = 0; i < kGroup; ++i) u[i] = w[i] >= 0.0f ? 1 : 0;  // sign(0) = +1
    return VBQ_OK;
  }
  const int m = (1 << (b - 1)) - 1;
  double amax = 0.0;
  for (int i = 0; i < kGroup; ++i) amax = std::max(amax, std::fabs((double)w[i]));
  uint16_t sb = to_fp16_bits(amax / m);
  if (!fp16_finite(sb)) return VBQ_ERR_SCALE_RANGE;
  *s_bits = sb;
  const double s = fp16_to_double(sb);  // codes use the stored scale
  const int off = 1 << (b - 1);
  for (int i = 0; i < kGroup; ++i) {
    double q = 0.0;
    if (s != 0.0) {
      q = std::nearbyint((double)w[i] / s);  // round half to even
      q = std::min<double>(std::max<double>(q, -m), m);
    }
    u[i] = (uint8_t)((int)q + off);
  }
  return VBQ_OK;
}

// Offset codes of already-quantized levels, with level-set validation.
inline vbq_status codes_of_levels(const int8_t* q, int b, uint8_t* u) {
  if (b == 1) {
    for (int i = 0; i < kGroup; ++i) {
      if (q[i] != 1 && q[i] != -1) return VBQ_ERR_CODE_RANGE;
      u[i] = (uint8_t)((q[i] + 1) / 2);
    }
    return VBQ_OK;
  }
  const int m = (1 << (b - 1)) - 1, off = 1 << (b - 1);
  for (int i = 0; i < kGroup; ++i) {
    if (q[i] < -m || q[i] > m) return VBQ_ERR_CODE_RANGE;
    u[i] = (uint8_t)(q[i] + off);
  }
  return VBQ_OK;
}

struct Source {
  const float* W = nullptr;         // vbq_pack
  const int8_t* q = nullptr;        // vbq_pack_codes
  const uint16_t* scales = nullptr;  // vbq_pack_codes
};

vbq_status pack_impl(int64_t N, int64_t K, const Source& src, const uint8_t* bits,
                     const vbq_pack_opts* opts, void* blob, size_t blob_bytes, vbq_desc* desc) {
  if (!bits || !blob || !desc) return VBQ_ERR_NULL;
  Geometry g;
  vbq_status st = make_geometry(N, K, opts, &g);
  if (st != VBQ_OK) return st;
  if (opts && opts->flags != 0) return VBQ_ERR_UNSUPPORTED;
  if ((uintptr_t)blob % 8 != 0) return VBQ_ERR_BUFFER;
  const uint32_t n_threads = opts ? opts->n_threads : 0;
  Counts cnt;
  if ((st = count_units(g, bits, n_threads, &cnt)) != VBQ_OK) return st;
  std::vector<uint32_t> starts;
  int64_t n_entries[4];
  if ((st = unit_starts(g, cnt, &starts, n_entries)) != VBQ_OK) return st;
  vbq_desc d;
  fill_desc_header(g, n_entries, &d);
  if (blob_bytes < d.total_bytes) return VBQ_ERR_BUFFER;

  uint8_t* base = (uint8_t*)blob;
  // zero the alignment padding between sections and after the last one
  uint64_t pos = 0;
  for (int s = 0; s < VBQ_NSECTIONS; ++s) {
    if (d.section_off[s] > pos) std::memset(base + pos, 0, d.section_off[s] - pos);
    pos = std::max<uint64_t>(pos, d.section_off[s] + d.section_len[s]);
  }
  if (d.total_bytes > pos) std::memset(base + pos, 0, d.total_bytes - pos);

  uint32_t* units = (uint32_t*)(base + d.section_off[VBQ_SEC_UNITS]);
  uint64_t* wmap = (uint64_t*)(base + d.section_off[VBQ_SEC_WMAP]);
  uint8_t* codes[4];
  uint16_t* scales[4];
  for (int c = 0; c < 4; ++c) {
    codes[c] = base + d.section_off[VBQ_SEC_CODES0 + c];
    scales[c] = (uint16_t*)(base + d.section_off[VBQ_SEC_SCALES0 + c]);
  }
  // unit table, including the totals row
  for (int64_t u = 0; u <= g.units; ++u) {
    uint32_t* row = units + (size_t)u * kUnitRowWords;
    for (int c = 0; c < 4; ++c) row[c] = starts[(size_t)u * 4 + c];
    row[4] = (uint32_t)(u < g.units ? wmap_offset(g, u / g.U, u % g.U) : g.wmap_words);
    row[5] = row[6] = row[7] = 0;
  }

  std::atomic<int> err{VBQ_OK};
  parallel_tiles(g.T, n_threads, [&](int64_t t) {
    if (err.load(std::memory_order_relaxed) != VBQ_OK) return;
    const int64_t rows = g.tile_rows(t);
    std::vector<uint64_t> planes;
    uint8_t u[kGroup];
    for (int64_t k = 0; k < g.U; ++k) {
      const int64_t unit = t * g.U + k;
      const int64_t W = g.unit_words(k), cols = g.chunk_cols(k), j0 = k * g.C;
      planes.assign((size_t)2 * W, 0);
      uint32_t next[4];
      for (int c = 0; c < 4; ++c) next[c] = starts[(size_t)unit * 4 + c];
      for (int64_t jl = 0; jl < cols; ++jl) {
        const int64_t j = j0 + jl;
        for (int64_t rl = 0; rl < rows; ++rl) {
          const int64_t r = t * g.R + rl;
          const int64_t p = jl * g.R + rl;
          const int b = bits[r * g.G + j];
          const int c = class_of_bits((uint8_t)b);
          if (c & 1) planes[(size_t)(p >> 6)] |= 1ull << (p & 63);
          if (c & 2) planes[(size_t)(W + (p >> 6))] |= 1ull << (p & 63);
          const uint32_t e = next[c]++;
          uint16_t sb;
          vbq_status gs;
          if (src.W) {
            gs = quantize_group(src.W + r * g.K + j * kGroup, b, u, &sb);
          } else {
            gs = codes_of_levels(src.q + r * g.K + j * kGroup, b, u);
            sb = src.scales[r * g.G + j];
            if (gs == VBQ_OK && !fp16_finite(sb)) gs = VBQ_ERR_NONFINITE;
            if (gs == VBQ_OK && (sb & 0x8000u)) gs = VBQ_ERR_SCALE_RANGE;
          }
          if (gs != VBQ_OK) {
            record_error(err, gs);
            return;
          }
          encode_record(u, b, codes[c] + (size_t)e * (8u << c));
          scales[c][e] = sb;
        }
      }
      std::memcpy(wmap + units[(size_t)unit * kUnitRowWords + 4], planes.data(), planes.size() * 8);
    }
  });
  if (err.load() != VBQ_OK) return (vbq_status)err.load();
  *desc = d;
  return VBQ_OK;
}

}  // namespace

extern "C" {

const char* vbq_status_string(vbq_status s) {
  switch (s) {
    case VBQ_OK: return "ok";
    case VBQ_ERR_NULL: return "null pointer";
    case VBQ_ERR_SHAPE: return "unsupported shape (need N >= 1, K >= 64, K % 64 == 0; 0 <= M <= 16)";
    case VBQ_ERR_BITS: return "bit-width outside {1,2,4,8}";
    case VBQ_ERR_CODE_RANGE: return "level outside the level set of its width";
    case VBQ_ERR_NONFINITE: return "non-finite weight or scale";
    case VBQ_ERR_SCALE_RANGE: return "scale overflows fp16 or is negative";
    case VBQ_ERR_BUFFER: return "buffer too small or misaligned";
    case VBQ_ERR_DESC: return "descriptor does not match this layout";
    case VBQ_ERR_HIP: return "HIP runtime error";
    case VBQ_ERR_UNSUPPORTED: return "unsupported option";
  }
  return "unknown status";
}

uint32_t vbq_layout_version(void) { return VBQ_LAYOUT_VERSION; }

vbq_status vbq_pack_size(int64_t N, int64_t K, const uint8_t* bits, const vbq_pack_opts* opts,
                         size_t* bytes, vbq_desc* desc_out) {
  if (!bits || !bytes) return VBQ_ERR_NULL;
  Geometry g;
  vbq_status st = make_geometry(N, K, opts, &g);
  if (st != VBQ_OK) return st;
  if (opts && opts->flags != 0) return VBQ_ERR_UNSUPPORTED;
  Counts cnt;
  if ((st = count_units(g, bits, opts ? opts->n_threads : 0, &cnt)) != VBQ_OK) return st;
  std::vector<uint32_t> starts;
  int64_t n_entries[4];
  if ((st = unit_starts(g, cnt, &starts, n_entries)) != VBQ_OK) return st;
  vbq_desc d;
  fill_desc_header(g, n_entries, &d);
  *bytes = (size_t)d.total_bytes;
  if (desc_out) *desc_out = d;
  return VBQ_OK;
}

vbq_status vbq_pack(int64_t N, int64_t K, const float* W, const uint8_t* bits,
                    const vbq_pack_opts* opts, void* blob, size_t blob_bytes, vbq_desc* desc) {
  if (!W) return VBQ_ERR_NULL;
  Source src;
  src.W = W;
  return pack_impl(N, K, src, bits, opts, blob, blob_bytes, desc);
}

vbq_status vbq_pack_codes(int64_t N, int64_t K, const int8_t* q, const uint16_t* scale_f16,
                          const uint8_t* bits, const vbq_pack_opts* opts, void* blob,
                          size_t blob_bytes, vbq_desc* desc) {
  if (!q || !scale_f16) return VBQ_ERR_NULL;
  Source src;
  src.q = q;
  src.scales = scale_f16;
  return pack_impl(N, K, src, bits, opts, blob, blob_bytes, desc);
}

namespace {

// Rows of each width in increasing row order, and the widths present.
vbq_status bucket_rows(int64_t N, const uint8_t* row_bits, std::vector<int64_t> rows[4]) {
  for (int64_t n = 0; n < N; ++n) {
    const int c = class_of_bits(row_bits[n]);
    if (c < 0) return VBQ_ERR_BITS;
    rows[c].push_back(n);
  }
  return VBQ_OK;
}

// Descriptor and byte size of one bucket (n rows of width 2^c, K columns).
vbq_status bucket_desc(int64_t n, int64_t K, int c, const vbq_pack_opts* opts, vbq_desc* d) {
  Geometry g;
  vbq_status st = make_geometry(n, K, opts, &g);
  if (st != VBQ_OK) return st;
  int64_t n_entries[4] = {0, 0, 0, 0};
  n_entries[c] = n * g.G;
  if (n_entries[c] > 0xFFFFFFFFll || g.wmap_words > 0xFFFFFFFFll) return VBQ_ERR_UNSUPPORTED;
  fill_desc_header(g, n_entries, d);
  return VBQ_OK;
}

}  // namespace

vbq_status vbq_pack_row_buckets_size(int64_t N, int64_t K, const uint8_t* row_bits, const vbq_pack_opts* opts,
                                     size_t* bytes, int32_t* n_buckets) {
  if (!row_bits || !bytes || !n_buckets) return VBQ_ERR_NULL;
  if (N < 1 || K < kGroup || K % kGroup != 0) return VBQ_ERR_SHAPE;
  if (opts && opts->flags != 0) return VBQ_ERR_UNSUPPORTED;
  std::vector<int64_t> rows[4];
  vbq_status st = bucket_rows(N, row_bits, rows);
  if (st != VBQ_OK) return st;
  uint64_t total = 0;
  int32_t nb = 0;
  for (int c = 0; c < 4; ++c) {
    if (rows[c].empty()) continue;
    vbq_desc d;
    if ((st = bucket_desc((int64_t)rows[c].size(), K, c, opts, &d)) != VBQ_OK) return st;
    total = align_up(total) + d.total_bytes;
    ++nb;
  }
  *bytes = (size_t)total;
  *n_buckets = nb;
  return VBQ_OK;
}

vbq_status vbq_pack_row_buckets(int64_t N, int64_t K, const int8_t* q, const uint16_t* scale_f16,
                                const uint8_t* row_bits, const vbq_pack_opts* opts, void* blob, size_t blob_bytes,
                                vbq_bucket buckets[VBQ_MAX_BUCKETS], int32_t* n_buckets, int32_t* row_index) {
  if (!q || !scale_f16 || !row_bits || !blob || !buckets || !n_buckets || !row_index) return VBQ_ERR_NULL;
  size_t need = 0;
  int32_t nb = 0;
  vbq_status st = vbq_pack_row_buckets_size(N, K, row_bits, opts, &need, &nb);
  if (st != VBQ_OK) return st;
  if ((uintptr_t)blob % 8 != 0 || blob_bytes < need) return VBQ_ERR_BUFFER;
  std::vector<int64_t> rows[4];
  bucket_rows(N, row_bits, rows);
  const int64_t G = K / kGroup;
  uint64_t off = 0;
  int64_t row_begin = 0;
  int32_t i = 0;
  std::vector<int8_t> qb;
  std::vector<uint16_t> sb;
  std::vector<uint8_t> bb;
  for (int c = 0; c < 4; ++c) {
    const int64_t n = (int64_t)rows[c].size();
    if (n == 0) continue;
    // the bucket's rows, gathered in order: the same input vbq_pack_codes
    // would get for these rows alone
    qb.resize((size_t)(n * K));
    sb.resize((size_t)(n * G));
    bb.assign((size_t)(n * G), (uint8_t)(1u << c));
    for (int64_t r = 0; r < n; ++r) {
      const int64_t src = rows[c][(size_t)r];
      std::memcpy(&qb[(size_t)(r * K)], q + src * K, (size_t)K);
      std::memcpy(&sb[(size_t)(r * G)], scale_f16 + src * G, (size_t)G * 2);
      row_index[row_begin + r] = (int32_t)src;
    }
    off = align_up(off);
    vbq_bucket& b = buckets[i];
    b = vbq_bucket{};
    b.bits = 1 << c;
    b.row_begin = row_begin;
    b.n_rows = n;
    b.blob_offset = off;
    Source src;
    src.q = qb.data();
    src.scales = sb.data();
    st = pack_impl(n, K, src, bb.data(), opts, (uint8_t*)blob + off, blob_bytes - off, &b.desc);
    if (st != VBQ_OK) return st;
    off += b.desc.total_bytes;
    row_begin += n;
    ++i;
  }
  *n_buckets = nb;
  return VBQ_OK;
}

vbq_status vbq_desc_check(const vbq_desc* d) {
  if (!d) return VBQ_ERR_NULL;
  if (d->magic != VBQ_MAGIC || d->version != VBQ_LAYOUT_VERSION || d->group != kGroup) return VBQ_ERR_DESC;
  vbq_pack_opts o{d->tile_rows, d->chunk_groups, 0, 0};
  Geometry g;
  if (make_geometry(d->N, d->K, &o, &g) != VBQ_OK) return VBQ_ERR_DESC;
  if (g.T != d->n_tiles || g.U != d->n_chunks || g.units != d->n_units) return VBQ_ERR_DESC;
  int64_t total = 0;
  for (int c = 0; c < 4; ++c) {
    if (d->n_entries[c] < 0) return VBQ_ERR_DESC;
    total += d->n_entries[c];
  }
  if (total != g.N * g.G) return VBQ_ERR_DESC;
  vbq_desc ref;
  fill_desc_header(g, d->n_entries, &ref);
  for (int s = 0; s < VBQ_NSECTIONS; ++s)
    if (ref.section_off[s] != d->section_off[s] || ref.section_len[s] != d->section_len[s]) return VBQ_ERR_DESC;
  if (ref.total_bytes != d->total_bytes) return VBQ_ERR_DESC;
  return VBQ_OK;
}

}  // extern "C"
