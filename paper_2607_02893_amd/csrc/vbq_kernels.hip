// Fused dequantize-and-multiply over packed variable-bit-width weights, for
// gfx950 (MI355X).  Paper section 6 ("Fused kernels over packed weights"):
// every group's packed codes are expanded in registers with the group scale
// and accumulated, so the full-precision matrix never exists in memory.
//
// Work decomposition (layout version 1, include/vbq.h):
//   * one workgroup (256 lanes, 4 wave64) owns a row tile and walks its
//     column-chunk units in order; inside a unit each wave owns a contiguous,
//     word-aligned slice of group columns and works alone until the end of
//     the tile (no workgroup barrier per unit);
//   * a wave finds where its entries of each width class start by counting
//     the class bits of the 2-bit width map before its slice, then rebuilds
//     in LDS the position of each of its entries (inverse ballot + mbcnt per
//     map word), so lanes can be handed 64 consecutive entries of ONE width;
//   * each lane decodes one 64-weight group with width-specific, branch-free
//     bit tricks: a masked field of codes, read as a pair of fp16 values, is a
//     power-of-two multiple of the codes, so v_dot2_f32_f16 multiplies two
//     weights by their activations in one instruction and the power of two is
//     folded in once per group;
//   * the offset of the offset-binary codes is removed with the group's
//     activation sum X_j = sum x: sum q x = sum u x - 2^(b-1) X_j (b >= 2),
//     sum q x = 2 sum u x - X_j (b = 1);
//   * per-group partial results go to LDS at their (row, column) position,
//     each wave sums its columns row by row, and the four per-wave row sums
//     are added in wave order: every sum has a fixed order, so results are
//     bitwise repeatable.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <cstdint>
#include <type_traits>

#include "vbq_layout.hpp"

namespace {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));


// One packed matrix on the device.  Every section is addressed by a 32-bit
// byte offset from the blob start (blobs are below 4 GiB), so loads use a
// scalar 64-bit base with a 32-bit per-lane offset.
struct DevMatrix {
  const uint8_t* blob;
  uint32_t off_units, off_wmap;
  uint32_t off_codes[4], off_scales[4];  // an empty class points at the unit table (offset 0)
  uint32_t n_entries[4];
  uint32_t wmap_words;   // 64-bit words in the width-map section
  uint32_t tile_words;   // width-map words of one row tile (all its units, both planes)
  uint32_t chunk_words;  // width-map words per plane of a unit with C columns
  int32_t N, K, G, R, C, T, U, logR;
};

template <typename T>
__device__ __forceinline__ T ld(const uint8_t* base, uint32_t off) {
  return *(const T*)(base + off);
}
template <typename T>
__device__ __forceinline__ T ld_nt(const uint8_t* base, uint32_t off) {
  return __builtin_nontemporal_load((const T*)(base + off));
}

struct MvArgs {
  DevMatrix m;
  const uint16_t* x;  // fp16 bits, row m at x + m*ldx
  void* y;            // row m at y + m*ldy elements (float, or fp16 bits when yf16)
  int64_t ldx, ldy;
  int32_t M;          // rows of x actually present (<= MT)
  int32_t S;          // slices per unit
  int32_t SW;         // group columns per window (LDS staging)
  int32_t yf16;       // 1: y holds fp16 (each fp32 result rounded to nearest even)
  // one activation row only: output row n goes to y[rows[n]] (skipped unless
  // 0 <= rows[n] < ylen); rows == nullptr writes y[n]
  const int32_t* rows;
  int64_t ylen;
};

// Element i of y as float, or as fp16 rounded to nearest even (the
// conversion instruction's default rounding).
__device__ __forceinline__ void store_y(void* y, size_t i, float v, int32_t f16) {
  if (f16)
    ((_Float16*)y)[i] = (_Float16)v;
  else
    ((float*)y)[i] = v;
}

// Stores output row n of a one-row product, through the row map if there is one.
__device__ __forceinline__ void store_row(const MvArgs& a, size_t n, float v) {
  if (a.rows == nullptr) {
    store_y(a.y, n, v, a.yf16);
  } else {
    const int64_t d = a.rows[n];
    if (d >= 0 && d < a.ylen) store_y(a.y, (size_t)d, v, a.yf16);
  }
}

__device__ __forceinline__ half2_t as_h2(uint32_t v) { return __builtin_bit_cast(half2_t, v); }

__device__ __forceinline__ float dot2(uint32_t codes, uint32_t xpair, float acc) {
  return __builtin_amdgcn_fdot2(as_h2(codes), as_h2(xpair), acc, false);
}

// dot2 into a fresh accumulator: the three-operand form with an inline zero
// (the accumulating two-operand form would need a register set to zero first)
__device__ __forceinline__ float dot2_first(uint32_t codes, uint32_t xpair) {
  float r;
  __asm__("v_dot2_f32_f16 %0, %1, %2, 0" : "=v"(r) : "v"(codes), "v"(xpair));
  return r;
}

__device__ __forceinline__ uint32_t shl(uint32_t w, int s) { return s >= 0 ? (w << s) : (w >> (-s)); }

// ---------------------------------------------------------------------------
// Decoder tables.  A field of width B at bit f*B of a word is moved by `shift`
// bits so that it sits at target bit t (of both half-words); masked, the pair
// of fp16 halves equals (u_even, u_odd) * value(t), where value(t) is the fp16
// value of one unit at bit t: 2^(t-24) inside the mantissa (t + B <= 10), and
// for a single bit in the exponent field 2^((1 << (t-10)) - 15).  Fields with
// the same t share an fp32 accumulator ("slot"); each slot is multiplied by
// 1/value(t) once per group.
//
// v_dot2_f32_f16 keeps a fixed window below the nominal exponent of its
// operands, so fields low in the mantissa of a subnormal lose precision
// (measured: up to 5e-5 of the sum of |terms| per instruction for 2-bit codes
// at bit 0, exact at bits 8-9).  1-bit codes use normal exponent bits and are
// exact; the multi-bit tables keep their fields in the upper mantissa bits.
// ---------------------------------------------------------------------------
struct Field {
  int shift, t;
};

template <int CLS>
struct Dec;

// 1-bit: 16 fields per word.  Targets 10..14 are the exponent bits (normal
// fp16 values 2^-14, 2^-13, 2^-11, 2^-7, 2); three shifts cover all fields.
template <>
struct Dec<0> {
  static constexpr int B = 1, kFields = 16, kSlots = 5;
  __device__ static constexpr Field field(int f) {
    return f >= 10 && f <= 14 ? Field{0, f} : f >= 5 && f <= 9 ? Field{5, f + 5} : f <= 4 ? Field{10, f + 10} : Field{-1, 14};
  }
  __device__ static constexpr int slot(int t) { return t - 10; }
  __device__ static constexpr float inv_value(int s) {  // 1 / value(10 + s)
    return s == 0 ? 16384.0f : s == 1 ? 8192.0f : s == 2 ? 2048.0f : s == 3 ? 128.0f : 0.5f;
  }
};

// 2-bit: 8 fields per word, moved to bits 4-5, 6-7, 8-9.
template <>
struct Dec<1> {
  static constexpr int B = 2, kFields = 8, kSlots = 3;
  __device__ static constexpr Field field(int f) {
    return f >= 2 && f <= 4 ? Field{0, 2 * f} : f <= 1 ? Field{6, 2 * f + 6} : Field{-6, 2 * f - 6};
  }
  __device__ static constexpr int slot(int t) { return (t - 4) / 2; }
  __device__ static constexpr float inv_value(int s) { return s == 0 ? 1048576.0f : s == 1 ? 262144.0f : 65536.0f; }
};

// 4-bit: 4 fields per word, all moved to bits 4-7.
template <>
struct Dec<2> {
  static constexpr int B = 4, kFields = 4, kSlots = 1;
  __device__ static constexpr Field field(int f) { return Field{4 - 4 * f, 4}; }
  __device__ static constexpr int slot(int) { return 0; }
  __device__ static constexpr float inv_value(int) { return 1048576.0f; }  // 2^20
};

// 8-bit: 2 fields per word, both at bits 0-7.
template <>
struct Dec<3> {
  static constexpr int B = 8, kFields = 2, kSlots = 1;
  __device__ static constexpr Field field(int f) { return Field{-8 * f, 0}; }
  __device__ static constexpr int slot(int) { return 0; }
  __device__ static constexpr float inv_value(int) { return 16777216.0f; }  // 2^24
};

// (The one- and two-row dot2 paths both use these tables; three or more rows
// go to the matrix-core kernel.)
template <int CLS, int MT>
using DecFor = Dec<CLS>;

// ---------------------------------------------------------------------------
// Index build: positions of each class's entries inside one unit.
// ---------------------------------------------------------------------------
struct UnitInfo {
  int j0, cols, rows, npos, W;  // first group column, columns, real rows, positions, words per plane
  uint32_t wmap_word;
};

// bit l set iff position 64w + l is a real position of the unit
__device__ __forceinline__ uint64_t valid_mask(int w, int npos, int R, int rows) {
  const int p0 = w * 64;
  const int left = npos - p0;
  uint64_t m = left >= 64 ? ~0ull : (left <= 0 ? 0ull : ((1ull << left) - 1));
  if (rows < R) {
    uint64_t v;
    if (R >= 64) {  // the word lies inside one column
      const int n = rows - (p0 & (R - 1));
      v = n <= 0 ? 0ull : (n >= 64 ? ~0ull : ((1ull << n) - 1));
    } else {
      const uint64_t pat = (1ull << rows) - 1;
      v = 0;
      for (int s = 0; s < 64; s += R) v |= pat << s;
    }
    m &= v;
  }
  return m;
}

__device__ __forceinline__ void class_masks(uint64_t p0, uint64_t p1, uint64_t v, uint64_t m[4]) {
  m[0] = ~p0 & ~p1 & v;
  m[1] = p0 & ~p1 & v;
  m[2] = ~p0 & p1 & v;
  m[3] = p0 & p1 & v;
}

__device__ __forceinline__ UnitInfo load_unit(const DevMatrix& mat, int t, int k) {
  UnitInfo u;
  u.j0 = k * mat.C;
  u.cols = min(mat.C, mat.G - u.j0);
  u.rows = min(mat.R, mat.N - t * mat.R);
  u.npos = u.cols * mat.R;
  u.W = (u.npos + 63) >> 6;
  // units are stored tile by tile and only a tile's last chunk can be narrower,
  // so the first map word follows from the geometry (no unit-table read on the
  // path to the first load)
  u.wmap_word = (uint32_t)t * mat.tile_words + 2u * (uint32_t)k * mat.chunk_words;
  return u;
}

__device__ __forceinline__ uint32_t lane_id() {
  return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}
// The lane index, recomputed where it is called: values derived from it are
// then not hoisted out of the work loop, where they would be held (or
// spilled) across the whole loop.
__device__ __forceinline__ uint32_t lane_id_here() {
  uint32_t l;
  __asm__ __volatile__("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)); }
__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }
// A wave-uniform value the compiler must treat as produced here (it cannot
// hoist its uses above this point).
__device__ __forceinline__ uint32_t opaque(uint32_t v) {
  __asm__ __volatile__("" : "+s"(v));
  return v;
}
__device__ __forceinline__ uint64_t opaque64(uint64_t v) {
  __asm__ __volatile__("" : "+s"(v));
  return v;
}

// ---------------------------------------------------------------------------
// Work split.  A workgroup of NW waves owns one row tile.  Each unit of the
// tile is cut into S slices (contiguous, width-map-word-aligned runs of group
// columns) and the U*S (unit, slice) items are dealt to the waves in turn.
// Positions are column-major, so a slice's positions are one contiguous run
// of the unit and its entries of each class are one contiguous run of that
// class's section: a wave finds where its runs start by counting the class
// bits of the width-map words before its slice.  Everything up to a per-wave
// row sum is wave-local (x staging, index, decode, partial sums), in a
// private LDS region of the wave, so no workgroup barrier is needed until the
// per-wave row sums are combined, in wave order, at the end of the tile.
// A slice is processed in windows of at most SW columns (one window for one
// activation row).
//
// x is staged column-contiguous with a 144-byte column stride (128 bytes of
// activations + 16 of padding), so an entry reads its column's 8 chunks at
// immediate offsets from one address and up to 8 distinct consecutive
// columns in one instruction fall on distinct banks.
// ---------------------------------------------------------------------------
constexpr int kXStride = 144;
constexpr int kXRegs = 4;  // 16-byte x chunks per lane for one row: windows of <= 32 columns

__host__ __device__ inline int align16(int v) { return (v + 15) & ~15; }

// Byte offsets inside one wave's LDS region (window of SW columns, R rows,
// MT activation rows).
struct WavePlan {
  int inv, xs, Xs, part, tab, bytes;
};

// tab_bytes: the 1-bit lookup tables of one group column (kLutBytes) for the
// one-width 1-bit kernel, else 0.  index: whether the wave builds a position
// index (one-width kernels find positions from the geometry and have none).
__host__ __device__ inline WavePlan wave_plan(int R, int SW, int MT, int tab_bytes = 0, bool index = true) {
  WavePlan p;
  int o = 0;
  p.tab = o;  o += tab_bytes;                      // 1-bit lookup tables (first: 256-byte aligned)
  p.inv = o;  o += index ? align16(SW * R * 2) : 0;  // uint16 local position of each entry
  p.xs = o;   o += MT * SW * kXStride;   // staged x
  p.Xs = o;   o += align16(MT * SW * 4); // per-column activation sums
  p.part = o; o += MT * SW * R * 4;      // per-entry partial products
  if (tab_bytes > 0) o = (o + 255) & ~255;  // keeps every wave's tables 256-byte aligned
  p.bytes = o;
  return p;
}

// Whole workgroup: NW row-sum arrays (MT*R floats each), then NW regions.
__host__ __device__ inline int mv_lds_bytes(int R, int SW, int MT, int NW, int tab_bytes = 0, bool index = true) {
  return NW * (MT * R * 4 + wave_plan(R, SW, MT, tab_bytes, index).bytes);
}

// Group columns per width-map word (1 when a column spans whole words).
__host__ __device__ inline int cols_per_word(int R) { return R >= 64 ? 1 : 64 / R; }

// Columns [cb, ce) of slice s of S of a unit with `cols` columns.
__host__ __device__ inline void slice_cols(int cols, int R, int s, int S, int& cb, int& ce) {
  const int cw = cols_per_word(R);
  const int per = ((cols + cw - 1) / cw + S - 1) / S;
  cb = min(cols, s * per * cw);
  ce = min(cols, (s + 1) * per * cw);
}

// Columns of the widest slice of a unit of C columns.
__host__ __device__ inline int max_slice_cols(int R, int C, int S) {
  int cb, ce;
  slice_cols(C, R, 0, S, cb, ce);
  return ce - cb;
}

__device__ __forceinline__ u32x4 lds_u32x4(uint32_t addr) {
  return *(const __attribute__((address_space(3))) u32x4*)(size_t)addr;
}
__device__ __forceinline__ float lds_f32(uint32_t addr) {
  return *(const __attribute__((address_space(3))) float*)(size_t)addr;
}
__device__ __forceinline__ void lds_store_f32(uint32_t addr, float v) {
  *(__attribute__((address_space(3))) float*)(size_t)addr = v;
}
__device__ __forceinline__ void lds_store_u32x4(uint32_t addr, u32x4 v) {
  *(__attribute__((address_space(3))) u32x4*)(size_t)addr = v;
}
__device__ __forceinline__ void lds_store_u16(uint32_t addr, uint16_t v) {
  *(__attribute__((address_space(3))) uint16_t*)(size_t)addr = v;
}
__device__ __forceinline__ int lds_u16(uint32_t addr) {
  return *(const __attribute__((address_space(3))) uint16_t*)(size_t)addr;
}
// Keeps the compiler from moving LDS accesses across phases of a wave that
// hand data between its lanes through LDS (a wave's LDS operations are
// executed in order, so no hardware wait is needed).
__device__ __forceinline__ void lds_phase() { __asm__ __volatile__("" ::: "memory"); }

__device__ __forceinline__ uint64_t read_lane64(uint64_t v, int l) {
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, l), hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}

// Width-map words 0 .. we-1 of the unit (both planes), lane l holding words
// l and l + 64.  Loads are unconditional, with indices clamped to the unit
// and to the section, so outstanding-load counts stay exact.
struct WmapRegs {
  uint64_t a0, a1;  // plane 0 / plane 1 of word l
  uint64_t b0, b1;  // plane 0 / plane 1 of word l + 64
};

__device__ __forceinline__ WmapRegs load_wmap(const DevMatrix& mat, const UnitInfo& u, int we, uint32_t lane) {
  const uint32_t last = mat.wmap_words - 1;
  const uint32_t top = (uint32_t)(max(we, 1) - 1);
  const uint32_t wa = min(lane, top), wb = min(lane + 64u, top);
  WmapRegs r;
  r.a0 = ld<uint64_t>(mat.blob, mat.off_wmap + 8u * min(u.wmap_word + wa, last));
  r.a1 = ld<uint64_t>(mat.blob, mat.off_wmap + 8u * min(u.wmap_word + (uint32_t)u.W + wa, last));
  r.b0 = ld<uint64_t>(mat.blob, mat.off_wmap + 8u * min(u.wmap_word + wb, last));
  r.b1 = ld<uint64_t>(mat.blob, mat.off_wmap + 8u * min(u.wmap_word + (uint32_t)u.W + wb, last));
  return r;
}

// Cross-lane moves on the VALU (DPP), no LDS round trip.  A lane whose
// source is outside its row of 16 reads 0.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xf, 0xf, true);
}
constexpr int kDppShr1 = 0x111, kDppShr2 = 0x112, kDppShr4 = 0x114, kDppShr8 = 0x118;
constexpr int kDppQuadXor1 = 0xB1, kDppQuadXor2 = 0x4E;  // quad_perm [1,0,3,2] and [2,3,0,1]

// v + (v of a neighbour lane), as floats
__device__ __forceinline__ float add_dpp_f32_quad_xor1(float s) {
  return s + __builtin_bit_cast(float, dpp<kDppQuadXor1>(__builtin_bit_cast(uint32_t, s)));
}
__device__ __forceinline__ float add_dpp_f32_quad_xor2(float s) {
  return s + __builtin_bit_cast(float, dpp<kDppQuadXor2>(__builtin_bit_cast(uint32_t, s)));
}
__device__ __forceinline__ float add_dpp_f32_shr4(float s) {
  return s + __builtin_bit_cast(float, dpp<kDppShr4>(__builtin_bit_cast(uint32_t, s)));
}


// Sum over the wave (integers): prefix sums inside each row of 16 lanes,
// then the four row totals.  The result is wave-uniform.
__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
  v += dpp<kDppShr1>(v);
  v += dpp<kDppShr2>(v);
  v += dpp<kDppShr4>(v);
  v += dpp<kDppShr8>(v);
  return __builtin_amdgcn_readlane(v, 15) + __builtin_amdgcn_readlane(v, 31) + __builtin_amdgcn_readlane(v, 47) +
         __builtin_amdgcn_readlane(v, 63);
}

// Class counts of words [0, wb) of the unit (where the window's runs start
// inside the unit's class runs) and of words [wb, we) (the window's runs).
struct WinCounts {
  uint32_t before[4], own[4];
};

__device__ __forceinline__ WinCounts window_counts(const WmapRegs& wr, const UnitInfo& u, int wb, int we, int R,
                                                   uint32_t lane) {
  uint32_t bef01 = 0, bef23 = 0, own01 = 0, own23 = 0;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int w = (int)lane + 64 * h;
    uint64_t m[4];
    class_masks(h ? wr.b0 : wr.a0, h ? wr.b1 : wr.a1, valid_mask(w, u.npos, R, u.rows), m);
    // packed 16-bit halves: a unit has at most 8192 positions
    const uint32_t c01 = (uint32_t)__popcll(m[0]) | ((uint32_t)__popcll(m[1]) << 16);
    const uint32_t c23 = (uint32_t)__popcll(m[2]) | ((uint32_t)__popcll(m[3]) << 16);
    if (w < wb) {
      bef01 += c01;
      bef23 += c23;
    } else if (w < we) {
      own01 += c01;
      own23 += c23;
    }
  }
  bef01 = wave_sum(bef01);
  bef23 = wave_sum(bef23);
  own01 = wave_sum(own01);
  own23 = wave_sum(own23);
  WinCounts wc;
  wc.before[0] = bef01 & 0xFFFF;
  wc.before[1] = bef01 >> 16;
  wc.before[2] = bef23 & 0xFFFF;
  wc.before[3] = bef23 >> 16;
  wc.own[0] = own01 & 0xFFFF;
  wc.own[1] = own01 >> 16;
  wc.own[2] = own23 & 0xFFFF;
  wc.own[3] = own23 >> 16;
  return wc;
}

// inv[k] (uint16, from byte offset `inv`) = window-local position of the
// k-th entry of the window, entries ordered by class, then by position.  One
// pass per width-map word, lane l taking position 64w + l: its rank inside
// its class is a masked bit count (mbcnt) of the class mask, its class
// selects among the four candidate slots (lane masks used directly as select
// conditions), and real positions write their slot.  No branch depends on
// the data.  Words whose 64 positions are all real (every word but a unit's
// last one, outside the ragged last tile) skip the validity masks.
// kFwd: write the other direction instead, fwd[pos] = (class << 14) | rank of
// the position inside its class (run[] then starts at 0 for every class).
template <bool kFull, bool kFwd = false>
__device__ __forceinline__ void index_word(uint64_t p0, uint64_t p1, uint64_t valid, uint32_t pos, uint32_t run[4],
                                           uint32_t inv) {
  uint64_t m[4];
  if constexpr (kFull) {
    m[0] = ~(p0 | p1);
    m[1] = p0 & ~p1;
    m[2] = p1 & ~p0;
    m[3] = p0 & p1;
  } else {
    class_masks(p0, p1, valid, m);
  }
  uint32_t slot[4];
#pragma unroll
  for (int c = 0; c < 4; ++c)
    slot[c] = __builtin_amdgcn_mbcnt_hi((uint32_t)(m[c] >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m[c], run[c]));
  uint32_t k = slot[3] | (kFwd ? 3u << 14 : 0u);
  k = __builtin_amdgcn_inverse_ballot_w64(m[2]) ? slot[2] | (kFwd ? 2u << 14 : 0u) : k;
  k = __builtin_amdgcn_inverse_ballot_w64(m[1]) ? slot[1] | (kFwd ? 1u << 14 : 0u) : k;
  k = __builtin_amdgcn_inverse_ballot_w64(m[0]) ? slot[0] : k;
  if constexpr (kFwd)
    lds_store_u16(inv + 2u * pos, (uint16_t)(__builtin_amdgcn_inverse_ballot_w64(valid) ? k : 0u));
  else if (kFull || __builtin_amdgcn_inverse_ballot_w64(valid))
    lds_store_u16(inv + 2u * k, (uint16_t)pos);
#pragma unroll
  for (int c = 0; c < 4; ++c) run[c] += (uint32_t)__popcll(m[c]);
}

template <bool kFwd = false>
__device__ __forceinline__ void build_index(const WmapRegs& wr, const UnitInfo& u, int wb, int we, int R,
                                            const WinCounts& wc, uint32_t inv, uint32_t lane) {
  uint32_t run[4];
  run[0] = 0;
  run[1] = kFwd ? 0u : wc.own[0];
  run[2] = kFwd ? 0u : run[1] + wc.own[1];
  run[3] = kFwd ? 0u : run[2] + wc.own[2];
  const int full_end = u.rows == R ? max(wb, min(we, u.npos >> 6)) : wb;
  const uint32_t pos0 = lane - (uint32_t)wb * 64u;
  // words held in lanes w (planes a0/a1) and w - 64 (planes b0/b1)
  for (int w = wb; w < min(full_end, 64); ++w)
    index_word<true, kFwd>(read_lane64(wr.a0, w), read_lane64(wr.a1, w), ~0ull, pos0 + 64u * w, run, inv);
  for (int w = max(wb, 64); w < full_end; ++w)
    index_word<true, kFwd>(read_lane64(wr.b0, w - 64), read_lane64(wr.b1, w - 64), ~0ull, pos0 + 64u * w, run, inv);
  for (int w = full_end; w < we; ++w) {
    const bool hi = w >= 64;
    index_word<false, kFwd>(read_lane64(hi ? wr.b0 : wr.a0, w & 63), read_lane64(hi ? wr.b1 : wr.a1, w & 63),
                      valid_mask(w, u.npos, R, u.rows), pos0 + 64u * w, run, inv);
  }
}

// ---------------------------------------------------------------------------
// Batches.  Every lane holds 32 bytes of codes per batch for widths 2, 4 and
// 8: E = 2 and 1 whole entries for widths 2 and 4, and half an entry for
// width 8 with one activation row (L = 2 lanes per entry: lanes 2j and 2j+1
// hold the low and high halves of one entry; several rows take whole 8-bit
// entries).  Width 1 takes E = 2 entries (16 bytes): with four (32 bytes) a
// wave keeps more bytes in flight, and every kernel got slower (the 9B-class
// step 1045 against 1070 us, the one-width 1-bit 1.46B-class step 557 against
// 570 us; one entry was slower again, 1058 and 603 us).  Slot i of batch b
// covers the run's entries (bE + i) * 64/L .. + 64/L - 1, one per lane (or
// lane pair), so every load instruction reads one contiguous span.
// ---------------------------------------------------------------------------
template <int CLS, int MT>
struct Batch {
  static constexpr int NW = 2 << CLS;                    // uint32 words per entry
  static constexpr int L = CLS == 3 && MT == 1 ? 2 : 1;  // lanes per entry
  static constexpr int E = CLS == 3 ? 1 : CLS == 0 ? 2 : 4 >> CLS;  // entry slots per lane
  static constexpr int LW = NW / L;                // words per lane per slot
  static constexpr int G = 64 / L;                 // entries per slot across the wave
  uint32_t w[E * LW];
  uint16_t s[E];
};

// Every lane always loads, whatever the run's length (lanes past the end
// re-read its last entry, clamped into the class section, and an empty run
// reads the section's first entry or, for an empty class, the unit table).
// Unconditional loads keep the number of outstanding loads the same on every
// path, so the compiler waits only for the batch it is about to decode and
// later batches stay in flight (a conditional load makes it wait for all).
template <int CLS, int MT>
__device__ __forceinline__ void load_batch(Batch<CLS, MT>& bt, const DevMatrix& mat, uint32_t start, int n, int b,
                                           uint32_t lane) {
  using BT = Batch<CLS, MT>;
  const uint32_t lim = max(mat.n_entries[CLS], 1u) - 1u;
  const uint32_t half = BT::L == 2 ? (lane & 1u) : 0u;
#pragma unroll
  for (int i = 0; i < BT::E; ++i) {
    const int e = max(min((b * BT::E + i) * BT::G + (int)(lane / BT::L), n - 1), 0);
    const uint32_t g = min(start + (uint32_t)e, lim);
    bt.s[i] = ld<uint16_t>(mat.blob, mat.off_scales[CLS] + 2u * g);
    const uint32_t off = mat.off_codes[CLS] + g * (4u * BT::NW) + half * (4u * BT::LW);
    if constexpr (BT::LW == 2) {
      const u32x2 v = ld_nt<u32x2>(mat.blob, off);
      bt.w[2 * i] = v.x;
      bt.w[2 * i + 1] = v.y;
    } else {
#pragma unroll
      for (int k = 0; k < BT::LW / 4; ++k) {
        const u32x4 v = ld_nt<u32x4>(mat.blob, off + 16u * k);
        bt.w[i * BT::LW + 4 * k] = v.x;
        bt.w[i * BT::LW + 4 * k + 1] = v.y;
        bt.w[i * BT::LW + 4 * k + 2] = v.z;
        bt.w[i * BT::LW + 4 * k + 3] = v.w;
      }
    }
  }
}

struct Win {  // LDS byte addresses of the wave's window buffers
  uint32_t xs, Xs, part, tab;
  uint32_t xstride_m;  // bytes between the staged x rows
  uint32_t part_m;     // bytes between the partial-product planes of two x rows
  int SW, logR;        // window columns (Xs row stride), log2 R
};

// First pair index (0..31) whose field lands in accumulator slot `sl`.
template <typename D>
__device__ constexpr int first_pair_of_slot(int sl) {
  for (int i = 0; i < 32; ++i)
    if (D::slot(D::field(i % D::kFields).t) == sl) return i;
  return 32;
}

// Decode one entry (64 weights) at window-local position p, reading the
// activations of the MT rows from LDS chunk by chunk, and write its partial
// product(s) to LDS.  Lanes past the end of a run hold a copy of the run's
// last entry (clamped loads), so they store the same value to the same place.
template <int CLS, int MT>
__device__ __forceinline__ void compute_entry(const uint32_t* w, uint16_t s_bits, int p, bool valid, uint32_t lane,
                                              const Win& wn) {
  using D = DecFor<CLS, MT>;
  constexpr int L = Batch<CLS, MT>::L;
  constexpr int NQ = 8 / L;  // x chunks (4 pairs each) this lane covers
  const int js = p >> wn.logR;
  // lane pairs of a half-entry class: the odd lane takes the high half
  const uint32_t xaddr = wn.xs + (uint32_t)__umul24((uint32_t)js, kXStride) + (L == 2 ? (lane & 1u) * 64u : 0u);
  // the column sums first: their LDS latency overlaps the products
  float Xm[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) Xm[m] = lds_f32(wn.Xs + 4u * (uint32_t)(m * wn.SW + js));
  float acc[MT][D::kSlots];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {  // local x chunk q holds pairs 4q..4q+3 of this lane's share
    u32x4 xv[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) xv[m] = lds_u32x4(xaddr + (uint32_t)m * wn.xstride_m + 16u * q);
#pragma unroll
    for (int c4 = 0; c4 < 4; ++c4) {
      const int i = 4 * q + c4;  // pair index within the lane's share (the field table repeats per word)
      const int wi = i / D::kFields, f = i % D::kFields;
      constexpr uint32_t one = (1u << D::B) - 1;
      const Field fd = D::field(f);
      const uint32_t mask = (one << fd.t) * 0x00010001u;
      const uint32_t v = shl(w[wi], fd.shift) & mask;
      const int sl = D::slot(fd.t);
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        if (i == first_pair_of_slot<D>(sl))  // resolved at compile time
          acc[m][sl] = MT <= 2 ? dot2_first(v, xv[m][c4]) : dot2(v, xv[m][c4], 0.0f);
        else
          acc[m][sl] = dot2(v, xv[m][c4], acc[m][sl]);
      }
    }
  }
  const float s = (float)__builtin_bit_cast(_Float16, s_bits);
  const uint32_t paddr = wn.part + 4u * (uint32_t)p;
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    float su = acc[m][0] * D::inv_value(0);
#pragma unroll
    for (int k = 1; k < D::kSlots; ++k) su = __builtin_fmaf(acc[m][k], D::inv_value(k), su);
    if constexpr (L == 2) su = add_dpp_f32_quad_xor1(su);  // both halves, the same sum in both lanes
    const float X = Xm[m];
    const float sq = CLS == 0 ? __builtin_fmaf(su, 2.0f, -X) : __builtin_fmaf(-(float)(1 << (D::B - 1)), X, su);
    // (several rows: skipping the duplicates keeps the register allocator's
    // scheduling regions small; one row stores them, with no branch)
    if (MT == 1 || valid) lds_store_f32(paddr + (uint32_t)m * wn.part_m, s * sq);
  }
}

// kUni: every entry of the window has width CLS, so the k-th one sits at the
// k-th real position: column k / rows, row k % rows (inv_c is then `rows`).
template <int CLS, int MT, bool kUni = false>
__device__ __forceinline__ void decode_batch(const Batch<CLS, MT>& bt, uint32_t inv_c, int n, int b, uint32_t lane,
                                             const Win& wn) {
  using BT = Batch<CLS, MT>;
  int p[BT::E];
#pragma unroll
  for (int i = 0; i < BT::E; ++i) {
    const int k = max(min((b * BT::E + i) * BT::G + (int)(lane / BT::L), n - 1), 0);
    if constexpr (kUni) {
      const int rows = (int)inv_c;
      p[i] = rows == (1 << wn.logR) ? k : (k / rows) * (1 << wn.logR) + k % rows;
    } else {
      p[i] = lds_u16(inv_c + 2u * (uint32_t)k);
    }
  }
#pragma unroll
  for (int i = 0; i < BT::E; ++i) {
    const int g0 = (b * BT::E + i) * BT::G;
    if (g0 < n)  // wave-uniform: whole slots past the end are skipped
      compute_entry<CLS, MT>(&bt.w[i * BT::LW], bt.s[i], p[i], g0 + (int)(lane / BT::L) < n, lane, wn);
    __builtin_amdgcn_sched_barrier(0);
  }
}

// ---------------------------------------------------------------------------
// 1-bit decode through lookup tables (one-width 1-bit matrices, full tiles of
// at least 64 rows, where a 64-entry slot is 64 rows of ONE group column).
//
// A 1-bit group's 64 codes are 16 nibbles: nibble n of word w holds the codes
// of weights i0 + 2t, t = 0..3, with i0 = 32w + 8(n & 3) + (n >> 2) (the even
// weights of the word's pairs in its low half-word, the odd ones in the high
// half-word).  For the slot's group column, table m = 8w + n holds the 16
// subset sums T_m[v] = sum over the set bits t of v of x[i0 + 2t] (fp32), so
// the sum of x over the group's 1-codes is sum_m T_m[nibble m]: 16 lookups
// instead of 32 masks and 32 two-term dot products.  The 16 entries of a
// table sit in 16 consecutive words, so the 64 lanes' lookups into one table
// never meet in a bank.  Then sum q x = 2 sum_{u=1} x - X_j as in the dot2
// path.  A table costs each lane one 16-byte read of x, a few adds and one
// 16-byte store, once per group column (every R/64 slots).
// ---------------------------------------------------------------------------
constexpr int kLutBytes = 16 * 16 * 4;  // 16 tables of 16 fp32 entries

// Lane l writes entries 4(l & 3) .. +3 of table l >> 2 for group column js.
__device__ __forceinline__ void build_lut(int js, const Win& wn, uint32_t lane) {
  const uint32_t m = lane >> 2, hi = lane & 3u;
  const uint32_t w = m >> 3, n = m & 7u, e = n >> 2;
  const uint32_t q = 4u * w + (n & 3u);  // x chunk of weights i0 .. i0 + 7
  const u32x4 c = lds_u32x4(wn.xs + (uint32_t)__umul24((uint32_t)js, kXStride) + 16u * q);
  const uint32_t sh = 16u * e;  // weight i0 + 2t is half e of dword t
  const float x0 = (float)__builtin_bit_cast(_Float16, (uint16_t)(c.x >> sh));
  const float x1 = (float)__builtin_bit_cast(_Float16, (uint16_t)(c.y >> sh));
  const float x2 = (float)__builtin_bit_cast(_Float16, (uint16_t)(c.z >> sh));
  const float x3 = (float)__builtin_bit_cast(_Float16, (uint16_t)(c.w >> sh));
  const float th = ((hi & 1u) ? x2 : 0.0f) + ((hi & 2u) ? x3 : 0.0f);  // bits 2, 3 of v = 4 hi + lo
  u32x4 t;
  t.x = __float_as_uint(th);
  t.y = __float_as_uint(th + x0);
  t.z = __float_as_uint(th + x1);
  t.w = __float_as_uint(th + (x0 + x1));
  lds_store_u32x4(wn.tab + 64u * m + 16u * hi, t);
}

// decode_batch for one-width 1-bit windows of full tiles with R >= 64: slot i
// of batch b is entries g0 .. g0 + 63, all in group column g0 / R, and the
// slot that starts a column first builds its tables.
//
// Table addresses: ta holds the tables' LDS base, which is 256-byte aligned,
// so its low byte is zero.  One SDWA AND per lookup writes nibble*4 into that
// byte and leaves the other three alone (dst_sel BYTE_0, UNUSED_PRESERVE),
// and the table's own offset 64 m rides in the LDS instruction: one VALU
// operation per lookup.  Byte k of w << 2, masked with 0x3C, is the low
// nibble of byte k of w times 4; byte k of w >> 2 gives the high nibble.
//
// kRowAcc (R == 64 and a run of whole slots): lane l's entry of every slot is
// row l, so each lane adds its slots' products to racc in column order (the
// order the per-entry partials would be summed in), with no partial-product
// store; otherwise the products go to the window's partial-product array.
template <int K>
__device__ __forceinline__ uint32_t lut_addr(uint32_t& ta, uint32_t shifted) {
  __asm__("v_and_b32_sdwa %0, 60, %1 dst_sel:BYTE_0 dst_unused:UNUSED_PRESERVE src0_sel:DWORD src1_sel:BYTE_%2"
          : "+v"(ta)
          : "v"(shifted), "n"(K));
  return ta;
}

template <bool kRowAcc>
__device__ __forceinline__ void decode_batch_lut(const Batch<0, 1>& bt, int n, int b, uint32_t lane, const Win& wn,
                                                 uint32_t (&ta)[4], float& racc) {
  constexpr int E = Batch<0, 1>::E;
#pragma unroll
  for (int i = 0; i < E; ++i) {
    const int g0 = (b * E + i) * 64;
    if (g0 < n) {  // wave-uniform: whole slots past the end are skipped
      const int js = g0 >> wn.logR;
      if ((g0 & ((1 << wn.logR) - 1)) == 0) {
        lds_phase();
        build_lut(js, wn, lane);
        lds_phase();
      }
      const float X = lds_f32(wn.Xs + 4u * (uint32_t)js);
      const uint32_t w0 = bt.w[2 * i], w1 = bt.w[2 * i + 1];
      const uint32_t sh[4] = {w0 << 2, w0 >> 2, w1 << 2, w1 >> 2};  // low / high nibbles of w0, w1
      float acc = 0.0f;
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        // table m = 8 (word) + nibble; nibble n of a word is the low (n even)
        // or high half of byte n >> 1
        uint32_t a;
        const uint32_t v = sh[2 * (m >> 3) + (m & 1)];
        switch ((m & 7) >> 1) {
          case 0: a = lut_addr<0>(ta[m & 3], v); break;
          case 1: a = lut_addr<1>(ta[m & 3], v); break;
          case 2: a = lut_addr<2>(ta[m & 3], v); break;
          default: a = lut_addr<3>(ta[m & 3], v); break;
        }
        const float t = lds_f32(a + 64u * (uint32_t)m);
        acc = m == 0 ? t : acc + t;
      }
      const float s = (float)__builtin_bit_cast(_Float16, bt.s[i]);
      const float v = s * __builtin_fmaf(acc, 2.0f, -X);
      if constexpr (kRowAcc) {
        racc += v;  // every slot is full (n is a multiple of 64)
      } else {
        // lanes past the end hold the run's last entry: same value, same place
        const int p = min(g0 + (int)lane, n - 1);
        lds_store_f32(wn.part + 4u * (uint32_t)p, v);
      }
      lds_phase();
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// run_class for the lookup-table decode (same double-buffered loop).
template <bool kRowAcc>
__device__ __forceinline__ void run_lut(const DevMatrix& mat, Batch<0, 1>& A, uint32_t start, int n, const Win& wn,
                                        uint32_t lane, float& racc) {
  constexpr int per_batch = Batch<0, 1>::E * Batch<0, 1>::G;
  const int nb = max(1, (n + per_batch - 1) / per_batch);
  uint32_t ta[4] = {wn.tab, wn.tab, wn.tab, wn.tab};
  if (nb == 1) {  // wave-uniform: no further batch, so no prefetch (each path keeps exact wait counts)
    decode_batch_lut<kRowAcc>(A, n, 0, lane, wn, ta, racc);
    return;
  }
  Batch<0, 1> B;
  for (int b = 0; b < nb; b += 2) {
    load_batch<0, 1>(B, mat, start, n, min(b + 1, nb - 1), lane);
    decode_batch_lut<kRowAcc>(A, n, b, lane, wn, ta, racc);
    if (b + 1 >= nb) break;
    load_batch<0, 1>(A, mat, start, n, min(b + 2, nb - 1), lane);
    decode_batch_lut<kRowAcc>(B, n, b + 1, lane, wn, ta, racc);
  }
}

// The n entries of class CLS of the window, starting at entry `start` of the
// class section.  Batch 0 is already in A (loaded with the other classes'
// first batches); the next batch is in flight while the current one is
// decoded.  The loop runs at least once and its loads are unconditional
// (past the last batch they repeat it), so the count of outstanding loads
// never depends on the data.

template <int CLS, int MT, bool kUni = false>
__device__ __forceinline__ void run_class(const DevMatrix& mat, Batch<CLS, MT>& A, uint32_t start, int n,
                                          uint32_t inv_c, const Win& wn, uint32_t lane) {
  constexpr int per_batch = Batch<CLS, MT>::E * Batch<CLS, MT>::G;
  const int nb = max(1, (n + per_batch - 1) / per_batch);
  if (MT == 1 && nb == 1) {  // wave-uniform: no further batch, so no prefetch (each path keeps exact wait counts)
    decode_batch<CLS, MT, kUni>(A, inv_c, n, 0, lane, wn);
    return;
  }
  Batch<CLS, MT> B;
  for (int b = 0; b < nb; b += 2) {
    load_batch<CLS, MT>(B, mat, start, n, min(b + 1, nb - 1), lane);
    decode_batch<CLS, MT, kUni>(A, inv_c, n, b, lane, wn);
    if (b + 1 >= nb) break;
    load_batch<CLS, MT>(A, mat, start, n, min(b + 2, nb - 1), lane);
    decode_batch<CLS, MT, kUni>(B, inv_c, n, b + 1, lane, wn);
  }
}

// x of one activation row for a window of `cols` <= 32 columns starting at
// group column j: lane l holds 16-byte chunks l, l + 64, ... (clamped loads).
struct XRegs {
  u32x4 v[kXRegs];
};

__device__ __forceinline__ void load_x1(const uint16_t* __restrict__ x, int j, int cols, XRegs& xr, uint32_t lane) {
  const int n = cols * 8;
  const uint8_t* xb = (const uint8_t*)x;
#pragma unroll
  for (int k = 0; k < kXRegs; ++k) {
    const int i = max(min((int)lane + 64 * k, n - 1), 0);
    xr.v[k] = ld<u32x4>(xb, 128u * (uint32_t)j + 16u * (uint32_t)i);  // chunk i of the window
  }
}

// Stores the chunks to LDS and writes each column's activation sum: every
// lane sums its chunk, the lanes of each quad add their sums pairwise
// (xor 1, then xor 2), and the last lane of the column's eight adds the
// first quad's sum to its own (a fixed order).
__device__ __forceinline__ void store_x1(int cols, const XRegs& xr, const Win& wn, uint32_t lane) {
  const int n = cols * 8;
  const uint32_t ones = 0x3C003C00u;  // (1.0, 1.0)
#pragma unroll
  for (int k = 0; k < kXRegs; ++k) {
    const int i = (int)lane + 64 * k;
    if (k * 64 < n) {  // wave-uniform
      const u32x4 v = xr.v[k];
      float sum = dot2(v.x, ones, 0.0f);
      sum = dot2(v.y, ones, sum);
      sum = dot2(v.z, ones, sum);
      sum = dot2(v.w, ones, sum);
      sum = add_dpp_f32_shr4(add_dpp_f32_quad_xor2(add_dpp_f32_quad_xor1(sum)));
      if (i < n) {
        lds_store_u32x4(wn.xs + (uint32_t)((i >> 3) * kXStride + (i & 7) * 16), v);
        if ((i & 7) == 7) lds_store_f32(wn.Xs + 4u * (uint32_t)(i >> 3), sum);
      }
    }
  }
}

// Several activation rows, as load_x1 / store_x1 row by row: every chunk's
// load is issued first (rows at or past M read row M-1 and are stored as
// zeros), so the staging costs one memory latency, not one per chunk.
template <int MT>
__device__ __forceinline__ void load_xm(const MvArgs& a, int j, int cols, XRegs (&xr)[MT], uint32_t lane) {
#pragma unroll
  for (int m = 0; m < MT; ++m) load_x1(a.x + (size_t)min(m, a.M - 1) * (size_t)a.ldx, j, cols, xr[m], lane);
}
template <int MT>
__device__ __forceinline__ void store_xm(const MvArgs& a, int cols, XRegs (&xr)[MT], const Win& wn, uint32_t lane) {
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    if (m >= a.M) {  // wave-uniform
#pragma unroll
      for (int k = 0; k < kXRegs; ++k) xr[m].v[k] = u32x4{0u, 0u, 0u, 0u};
    }
    Win w = wn;
    w.xs = wn.xs + (uint32_t)m * wn.xstride_m;
    w.Xs = wn.Xs + 4u * (uint32_t)(m * wn.SW);
    store_x1(cols, xr[m], w, lane);
  }
}

// Adds the window's row sums (columns 0..cols-1 in order) to the wave's row
// sums: lane l owns the (row, x-row) slots l, l + 64, ...
template <int MT>
__device__ __forceinline__ void reduce_window(const Win& wn, int R, int cols, int rows, uint32_t ysum,
                                              uint32_t lane) {
  for (int slot = (int)lane; slot < MT * R; slot += 64) {
    const int m = slot >> wn.logR, r = slot & (R - 1);
    if (r >= rows) continue;
    const uint32_t base = wn.part + (uint32_t)m * wn.part_m + 4u * (uint32_t)r;
    float acc = 0.0f;
    int j = 0;
    for (; j + 8 <= cols; j += 8) {
      float v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = lds_f32(base + 4u * (uint32_t)((j + k) * R));
#pragma unroll
      for (int k = 0; k < 8; ++k) acc += v[k];
    }
    for (; j < cols; ++j) acc += lds_f32(base + 4u * (uint32_t)(j * R));
    const uint32_t ya = ysum + 4u * (uint32_t)slot;
    lds_store_f32(ya, lds_f32(ya) + acc);
  }
}

// Start of unit `unit`'s class-c run in the class section.  The unit table
// is the blob's first section (offset 0, checked on the host).
__device__ __forceinline__ uint32_t class_start(const DevMatrix& mat, int unit, int c) {
  return ld<uint32_t>(mat.blob, 4u * ((uint32_t)unit * vbq::kUnitRowWords + c));
}
// Rows `unit` and `unit` + 1 of the unit table (one 64-byte load; the table
// has n_units + 1 rows): .s0123 are the unit's class-run starts, .s89ab the
// next unit's.
typedef uint32_t u32x16 __attribute__((ext_vector_type(16)));
__device__ __forceinline__ u32x16 unit_rows(const DevMatrix& mat, int unit) {
  return ld<u32x16>(mat.blob, 4u * (uint32_t)unit * vbq::kUnitRowWords);
}

// The same two rows read through the vector memory path (lane l reads word
// l & 15, then the 16 words are moved to scalar registers).  Measured against
// the scalar load: faster in the matrix-core kernel (1.46B-class M = 4: Q|K|V
// 7.74 -> 7.50 us a launch) and in the 16-wave pair kernel (9B-class down
// 8.37 -> 8.19 us), slower in the 8-wave pair kernel (1.46B-class step 660 ->
// 675 us), so only those two use it.
__device__ __forceinline__ u32x16 unit_rows_vec(const DevMatrix& mat, int unit) {
  const uint32_t l = __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)) & 15u;
  const uint32_t v = ld<uint32_t>(mat.blob, 4u * ((uint32_t)unit * vbq::kUnitRowWords + l));
  u32x16 r;
#pragma unroll
  for (int i = 0; i < 16; ++i) r[i] = __builtin_amdgcn_readlane(v, i);
  return r;
}

// Entries of a run that stay inside the class section (a malformed blob can
// make the width map and the unit table disagree).
__device__ __forceinline__ int clamp_run(const DevMatrix& mat, int c, uint32_t start, uint32_t n) {
  const uint32_t lim = mat.n_entries[c];
  return start >= lim ? 0 : (int)min(n, lim - start);
}

// One row tile of a one-width matrix (class UNI, one activation row): the
// workgroup's NW waves take the tile's items (unit slices) in turn, decode
// them and add their row sums, then the workgroup adds the waves' sums and
// writes the tile's rows.  Every group has width class UNI, so entries sit at
// consecutive real positions: no width map, no class counts, no index, and a
// unit's first entry follows from the geometry.  Shared by vbq_mv_kernel and
// the all-buckets kernel.
template <int NW, int UNI>
__device__ __forceinline__ void uniform_tile(const DevMatrix& mat, const MvArgs& a, int t, int S, int SW) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int R = mat.R;
  const uint32_t lds0 = (uint32_t)(size_t)(__attribute__((address_space(3))) uint8_t*)smem;
  const uint32_t lane = lane_id();
  const int wave = wave_id();
  const WavePlan P = wave_plan(R, SW, 1, UNI == 0 ? kLutBytes : 0, false);
  const uint32_t ysum = lds0 + (uint32_t)(wave * R * 4);
  const uint32_t region = lds0 + (uint32_t)(NW * R * 4 + wave * P.bytes);
  Win wn;
  wn.xs = region + P.xs;
  wn.Xs = region + P.Xs;
  wn.part = region + P.part;
  wn.tab = region + P.tab;
  wn.xstride_m = (uint32_t)(SW * kXStride);
  wn.part_m = (uint32_t)(SW * R * 4);
  wn.SW = SW;
  wn.logR = mat.logR;
  for (int i = (int)lane; i < R; i += 64) lds_store_f32(ysum + 4u * i, 0.0f);

  for (int item = wave; item < mat.U * S; item += NW) {
    const uint32_t lane = lane_id_here();
    const int k = item / S, sl = item - k * S;
    const UnitInfo u = load_unit(mat, t, k);
    int cb, ce;
    slice_cols(u.cols, R, sl, S, cb, ce);
    if (cb >= ce) continue;  // wave-uniform: an empty slice
    XRegs xr;
    load_x1(a.x, u.j0 + cb, ce - cb, xr, lane);
    // all tiles above this one are full: R*G entries each; this tile's units
    // hold C*rows entries each
    const uint32_t first = (uint32_t)t * (uint32_t)(R * mat.G) + (uint32_t)(u.j0 + cb) * (uint32_t)u.rows;
    const int cols = ce - cb;
    const int n = clamp_run(mat, UNI, first, (uint32_t)(cols * u.rows));
    Batch<UNI, 1> A;
    load_batch<UNI, 1>(A, mat, first, n, 0, lane);
    store_x1(cols, xr, wn, lane);
    lds_phase();
    if constexpr (UNI == 0) {
      // the table addressing needs the tables on a 256-byte boundary (the
      // dynamic LDS starts at 0 and the wave regions are multiples of 256
      // bytes; should that ever not hold, the dot2 decode runs instead)
      const bool tab_ok = (wn.tab & 255u) == 0u;
      // wave-uniform: lane l holds row l of every slot, and every slot is
      // whole (a run cut short by a malformed blob takes the path below)
      if (tab_ok && R == 64 && u.rows == 64 && n == cols * 64) {
        float racc = 0.0f;
        run_lut<true>(mat, A, first, n, wn, lane, racc);
        lds_phase();
        const uint32_t ya = ysum + 4u * lane;
        lds_store_f32(ya, lds_f32(ya) + racc);
        lds_phase();
        continue;
      }
      if (tab_ok && R > 64 && u.rows == R) {  // wave-uniform: slots of one column each
        float unused = 0.0f;
        run_lut<false>(mat, A, first, n, wn, lane, unused);
      } else {
        run_class<UNI, 1, true>(mat, A, first, n, (uint32_t)u.rows, wn, lane);
      }
    } else {
      run_class<UNI, 1, true>(mat, A, first, n, (uint32_t)u.rows, wn, lane);
    }
    lds_phase();
    reduce_window<1>(wn, R, cols, u.rows, ysum, lane);
    lds_phase();
  }
  __syncthreads();
  const int rows = min(R, mat.N - t * R);
  for (int r = threadIdx.x; r < rows; r += NW * 64) {
    float tot = 0.0f;
#pragma unroll
    for (int w2 = 0; w2 < NW; ++w2) tot += lds_f32(lds0 + 4u * (uint32_t)(w2 * R + r));
    store_row(a, (size_t)t * R + r, tot);
  }
}

// One activation row keeps 4 waves per SIMD (at most 128 VGPRs); more rows
// trade occupancy for registers.
//
// The values the first memory accesses depend on come as separate leading
// arguments, which the command processor can place in SGPRs before the wave
// starts (kernel-argument preloading), so the first loads do not wait for a
// kernel-argument fetch.  geo packs R (9 bits), C (8), log2 R (4) and S (8);
// sw_m packs SW (16) and M (16).  (At most 16 SGPRs can be preloaded, two
// of which hold the kernel-argument pointer: these eleven take 13.)
//
// UNI >= 0: every group of the matrix has width class UNI (a uniform "recipe"
// matrix, one row only).  Entries then sit at consecutive real positions, so
// the width map, the class counts and the index are not needed, and a unit's
// first entry follows from the geometry.  The three width-map arguments then
// carry the class's code offset, scale offset and entry count instead, which
// the first code loads need.
template <int MT, int NW, int UNI = -1>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(MT == 1 ? 4 : 2))) void vbq_mv_kernel(
    const uint16_t* __restrict__ x, const uint8_t* __restrict__ blob, uint32_t off_wmap, uint32_t tile_words,
    uint32_t chunk_words, uint32_t wmap_words, int32_t G, int32_t N, uint32_t geo, int32_t U, uint32_t sw_m,
    MvArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  DevMatrix mat = a.m;
  mat.blob = blob;
  if constexpr (UNI >= 0) {
    // no width map: these three carry the one class's code and scale offsets
    // and entry count, which the first code loads need
    mat.off_codes[UNI] = off_wmap;
    mat.off_scales[UNI] = tile_words;
    mat.n_entries[UNI] = chunk_words;
  } else {
    mat.off_wmap = off_wmap;
    mat.tile_words = tile_words;
    mat.chunk_words = chunk_words;
  }
  mat.wmap_words = wmap_words;
  mat.G = G;
  mat.N = N;
  mat.U = U;
  mat.R = (int)(geo & 0x1FF);
  mat.C = (int)((geo >> 9) & 0xFF);
  mat.logR = (int)((geo >> 17) & 0xF);
  a.x = x;
  a.M = (int)(sw_m >> 16);
  const int R = mat.R, SW = (int)(sw_m & 0xFFFF), S = (int)(geo >> 21);
  if constexpr (UNI >= 0) {
    static_assert(MT == 1, "one-width matrices take one activation row");
    uniform_tile<NW, UNI>(mat, a, blockIdx.x, S, SW);  // one row tile per workgroup
  } else {
    const uint32_t lds0 = (uint32_t)(size_t)(__attribute__((address_space(3))) uint8_t*)smem;
    const uint32_t lane = lane_id();
    const int wave = wave_id();
    const int t = blockIdx.x;  // one row tile per workgroup
    const int NS = MT * R;
    const WavePlan P = wave_plan(R, SW, MT);
    const uint32_t ysum = lds0 + (uint32_t)(wave * NS * 4);
    const uint32_t region = lds0 + (uint32_t)(NW * NS * 4 + wave * P.bytes);
    Win wn;
    wn.xs = region + P.xs;
    wn.Xs = region + P.Xs;
    wn.part = region + P.part;
    wn.tab = region + P.tab;
    wn.xstride_m = (uint32_t)(SW * kXStride);
    wn.part_m = (uint32_t)(SW * R * 4);
    wn.SW = SW;
    wn.logR = mat.logR;
    const uint32_t inv = region + P.inv;
    for (int i = (int)lane; i < NS; i += 64) lds_store_f32(ysum + 4u * i, 0.0f);

    for (int item = wave; item < mat.U * S; item += NW) {
      const uint32_t lane = lane_id_here();
      const int k = item / S, sl = item - k * S;
      const UnitInfo u = load_unit(mat, t, k);
      const int unit = t * mat.U + k;
      int cb, ce;
      slice_cols(u.cols, R, sl, S, cb, ce);
      if (cb >= ce) continue;  // wave-uniform: an empty slice
      // one or two rows: a wave's set-up (x, the map, the first code loads and
      // the index) runs at a raised issue priority, so a wave that has just
      // started gets its loads out ahead of the decode of the waves around it
      // (9B-class LM head: 38.8 -> 37.7 us a launch in the step; two rows:
      // 72.2 -> 71.0 us, the 9B-class down 17.6 -> 17.4 us)
      if (MT <= 2) __builtin_amdgcn_s_setprio(1);
      const int slice_we = (ce * R + 63) >> 6;
      XRegs xr;
      if constexpr (MT == 1) load_x1(a.x, u.j0 + cb, ce - cb, xr, lane);  // with the map: one latency
      // A whole-unit item (one slice per unit) reads where its class runs start
      // and how long they are from the unit table (rows u and u + 1): no class
      // counts, and its code loads do not wait for the width map.
      const bool whole = MT == 1 && S == 1;  // wave-uniform
      const u32x16 rows2 = unit_rows(mat, unit);
      const u32x4 erow = rows2.s0123, enext = rows2.s89ab;
      const uint32_t ustart[4] = {erow.x, erow.y, erow.z, erow.w};
      const WmapRegs wr = load_wmap(mat, u, slice_we, lane);
      // The class sections' offsets and sizes come from the kernel-argument
      // block (not preloaded): read them only now, so that the loads above do
      // not wait for that block (it would otherwise be read, and waited for,
      // before the work loop).
      lds_phase();
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        mat.off_codes[c] = opaque(mat.off_codes[c]);
        mat.off_scales[c] = opaque(mat.off_scales[c]);
        mat.n_entries[c] = opaque(mat.n_entries[c]);
      }
      auto window = [&](int c0, int c1) __attribute__((always_inline)) {
        const int cols = c1 - c0;
        const int wb = (c0 * R) >> 6, we = (c1 * R + 63) >> 6;
        const bool unit_window = whole && c0 == cb && c1 == ce;  // wave-uniform
        WinCounts wc;
        if (unit_window) {
          const u32x4 own = enext - erow;
          wc.own[0] = own.x;
          wc.own[1] = own.y;
          wc.own[2] = own.z;
          wc.own[3] = own.w;
#pragma unroll
          for (int c = 0; c < 4; ++c) wc.before[c] = 0u;
        } else {
          wc = window_counts(wr, u, wb, we, R, lane);
        }
        XRegs xrm[MT > 1 ? MT : 1];
        if constexpr (MT > 1) load_xm<MT>(a, u.j0 + c0, cols, xrm, lane);  // (several rows: per window)
        uint32_t start[4], seg[4];
        int n[4];
        uint32_t o = 0;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          start[c] = ustart[c] + wc.before[c];
          n[c] = clamp_run(mat, c, start[c], wc.own[c]);
          seg[c] = inv + 2u * o;
          o += wc.own[c];
        }
        // the 1- and 2-bit runs' first batches are in flight while x is stored
        // and the index is built (and, for several rows, x is staged); the 4-
        // and 8-bit runs' first batches go out one run ahead of their decode
        // (all four at once made every wave's chain longer: the 9B-class LM
        // head took 40.6-41.3 us against 39.7-39.9, at 128 VGPRs against 107)
        Batch<0, MT> A0;
        Batch<1, MT> A1;
        Batch<2, MT> A2;
        Batch<3, MT> A3;
        load_batch<0, MT>(A0, mat, start[0], n[0], 0, lane);
        load_batch<1, MT>(A1, mat, start[1], n[1], 0, lane);
        // one row: x arrived with the map and goes to LDS now
        if constexpr (MT == 1) store_x1(cols, xr, wn, lane);
        build_index(wr, u, wb, we, R, wc, inv, lane);
        if constexpr (MT > 1) store_xm<MT>(a, cols, xrm, wn, lane);
        lds_phase();
        if (MT <= 2) __builtin_amdgcn_s_setprio(0);
        run_class<0, MT>(mat, A0, start[0], n[0], seg[0], wn, lane);
        load_batch<2, MT>(A2, mat, start[2], n[2], 0, lane);
        run_class<1, MT>(mat, A1, start[1], n[1], seg[1], wn, lane);
        load_batch<3, MT>(A3, mat, start[3], n[3], 0, lane);
        run_class<2, MT>(mat, A2, start[2], n[2], seg[2], wn, lane);
        run_class<3, MT>(mat, A3, start[3], n[3], seg[3], wn, lane);
        lds_phase();
        reduce_window<MT>(wn, R, cols, u.rows, ysum, lane);
        lds_phase();
      };
      if constexpr (MT == 1) {
        window(cb, ce);  // one row: the window is the whole slice
      } else {
        for (int c0 = cb; c0 < ce; c0 += SW) window(c0, min(ce, c0 + SW));
      }
    }
    __syncthreads();
    const int rows = min(R, mat.N - t * R);
    for (int slot = threadIdx.x; slot < NS; slot += NW * 64) {
      const int m = slot >> mat.logR, r = slot & (R - 1);
      if (m < a.M && r < rows) {
        float tot = 0.0f;
#pragma unroll
        for (int w2 = 0; w2 < NW; ++w2) tot += lds_f32(lds0 + 4u * (uint32_t)(w2 * NS + slot));
        if (MT == 1)
          store_row(a, (size_t)t * R + r, tot);
        else
          store_y(a.y, m * a.ldy + (size_t)t * R + r, tot, a.yf16);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Every row bucket of a bucketed matrix in one launch (one-width buckets, one
// activation row).  Workgroups [tile0[b], tile0[b + 1]) take bucket b's row
// tiles; each runs uniform_tile for its bucket's width class, so a tile's
// arithmetic is that of the bucket's own vbq_gemv_rows launch.  The buckets
// run side by side instead of one after another.
// ---------------------------------------------------------------------------
struct BucketsArgs {
  DevMatrix m[VBQ_MAX_BUCKETS];
  const int32_t* rows[VBQ_MAX_BUCKETS];  // output row of each bucket row
  int32_t tile0[VBQ_MAX_BUCKETS];        // first workgroup of each bucket
  int32_t cls[VBQ_MAX_BUCKETS];          // width class (log2 bits)
  int32_t S[VBQ_MAX_BUCKETS];            // slices per unit
  int32_t SW[VBQ_MAX_BUCKETS];           // window columns
  int32_t n;                             // buckets
  int32_t yf16;
  const uint16_t* x;
  void* y;
  int64_t ylen;
};

template <int NW>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(4))) void vbq_buckets_kernel(BucketsArgs ba) {
  int b = 0;
#pragma unroll
  for (int i = 1; i < VBQ_MAX_BUCKETS; ++i)
    if (i < ba.n && (int)blockIdx.x >= ba.tile0[i]) b = i;
  MvArgs a;
  a.m = ba.m[b];
  a.x = ba.x;
  a.y = ba.y;
  a.ldx = 0;
  a.ldy = 0;
  a.M = 1;
  a.S = ba.S[b];
  a.SW = ba.SW[b];
  a.yf16 = ba.yf16;
  a.rows = ba.rows[b];
  a.ylen = ba.ylen;
  const int t = (int)blockIdx.x - ba.tile0[b];
  switch (ba.cls[b]) {
    case 0: uniform_tile<NW, 0>(a.m, a, t, a.S, a.SW); break;
    case 1: uniform_tile<NW, 1>(a.m, a, t, a.S, a.SW); break;
    case 2: uniform_tile<NW, 2>(a.m, a, t, a.S, a.SW); break;
    default: uniform_tile<NW, 3>(a.m, a, t, a.S, a.SW); break;
  }
}

// ---------------------------------------------------------------------------
// Two waves per unit (one or two activation rows, mixed widths, small matrices).
//
// With one wave per unit a small matrix leaves each SIMD one or two waves,
// and every wave runs its index build and its four class runs one after the
// other, each a chain of LDS round trips.  Here a pair of waves shares the
// unit: role 0 loads the width map, builds the index and decodes the 1- and
// 8-bit runs; role 1 loads x, stages it and decodes the 2- and 4-bit runs.
// Both read the unit's class runs from the unit table (rows u and u + 1), so
// both issue their first code loads at once.  Workgroup barriers separate
// the set-up, the decode and the row reduction.
//
// A wave's class runs follow one another, and every run after the first
// batch waits on memory for each further batch (a run of a few batches of
// short decodes hides little of that wait), so what bounds a role is mostly
// its number of batches.  A unit's short runs (2-, 4- and 8-bit, about two
// batches each) therefore go two to role 1 and one to role 0, beside the
// long 1-bit run whose decode covers its own next loads: measured against
// all three on role 1, the 9B-class step took 1075-1080 us instead of 1102,
// the 1.46B-class step 682 instead of 723 us.
//
// The roles do unequal VALU work (the 1-bit run is most of the entries), and
// a workgroup's waves are dealt to the CU's four SIMDs in turn, so with pairs
// (2k, 2k + 1) a CU holding one workgroup puts every role-0 wave on two SIMDs
// and every role-1 wave on the other two (measured with the hardware ids of
// each wave).  When more than half of the pairs have a unit, pair k is waves
// k and k + NW/2 instead: both land on one SIMD, so every SIMD carries both
// roles.  With fewer units, (2k, 2k + 1) spreads the busy waves over more SIMDs.
//
// MT = 2 activation rows uses the same split (x of both rows loaded by role 1
// with the map and every class's first batch loaded before the first barrier,
// as for one row), in 8-wave workgroups only: two rows need more than the 128
// registers a wave of a 16-wave workgroup can have.
// ---------------------------------------------------------------------------
template <int NW, int MT>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(MT == 1 ? 4 : 2))) void vbq_mv_pair_kernel(
    const uint16_t* __restrict__ x, const uint8_t* __restrict__ blob, uint32_t off_wmap, uint32_t tile_words,
    uint32_t chunk_words, uint32_t wmap_words, int32_t G, int32_t N, uint32_t geo, int32_t U, uint32_t sw_m,
    MvArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  constexpr int NP = NW / 2;  // wave pairs: one unit each
  DevMatrix mat = a.m;
  mat.blob = blob;
  mat.off_wmap = off_wmap;
  mat.tile_words = tile_words;
  mat.chunk_words = chunk_words;
  mat.wmap_words = wmap_words;
  mat.G = G;
  mat.N = N;
  mat.U = U;
  mat.R = (int)(geo & 0x1FF);
  mat.C = (int)((geo >> 9) & 0xFF);
  mat.logR = (int)((geo >> 17) & 0xF);
  a.x = x;
  a.M = (int)(sw_m >> 16);
  const int R = mat.R, SW = (int)(sw_m & 0xFFFF);
  const uint32_t lds0 = (uint32_t)(size_t)(__attribute__((address_space(3))) uint8_t*)smem;
  const uint32_t lane = lane_id();
  const int wave = wave_id();
  const bool mix = U > NP / 2;  // wave-uniform
  const int pair = mix ? wave % NP : wave >> 1, role = mix ? wave / NP : wave & 1;
  const int t = blockIdx.x;
  const WavePlan P = wave_plan(R, SW, MT);
  // one row: role 0 carries the longer chain (the map, the index, then the
  // 1-bit run, the longest), so its waves issue first wherever both roles
  // are ready: 9B-class step 1045 -> 1019 us, 1.46B-class 676 -> 661 us.  The
  // same priority for the decode alone changed nothing (the set-up is what it
  // shortens), and at two rows it made the 1.46B-class step 0.5% slower.
  if (MT == 1 && role == 0) __builtin_amdgcn_s_setprio(1);
  const uint32_t ysum = lds0 + (uint32_t)(pair * MT * R * 4);
  const uint32_t region = lds0 + (uint32_t)(NP * MT * R * 4 + pair * P.bytes);
  Win wn;
  wn.xs = region + P.xs;
  wn.Xs = region + P.Xs;
  wn.part = region + P.part;
  wn.xstride_m = (uint32_t)(SW * kXStride);
  wn.part_m = (uint32_t)(SW * R * 4);
  wn.SW = SW;
  wn.logR = mat.logR;
  const uint32_t inv = region + P.inv;
  if (role == 0)
    for (int i = (int)lane; i < MT * R; i += 64) lds_store_f32(ysum + 4u * i, 0.0f);

  const bool active = pair < mat.U;  // wave-uniform
  const UnitInfo u = load_unit(mat, t, active ? pair : 0);
  const int unit = t * mat.U + (active ? pair : 0);
  Batch<0, MT> A0;
  Batch<1, MT> A1;
  Batch<2, MT> A2;
  Batch<3, MT> A3;
  uint32_t start[4], seg[4];
  int n[4];
  if (active) {
    WmapRegs wr;
    XRegs xr;
    XRegs xrm[MT > 1 ? MT : 1];
    if (role == 0)
      wr = load_wmap(mat, u, u.W, lane);
    else if constexpr (MT == 1)
      load_x1(x, u.j0, u.cols, xr, lane);
    else
      load_xm<MT>(a, u.j0, u.cols, xrm, lane);  // (several rows: with the map, like one row)
    const u32x16 rows2 = NW == 16 ? unit_rows_vec(mat, unit) : unit_rows(mat, unit);
    const u32x4 erow = rows2.s0123, own = rows2.s89ab - rows2.s0123;
    // (the class sections' offsets come from the kernel-argument block: read
    // them only after the loads above are issued)
    lds_phase();
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      mat.off_codes[c] = opaque(mat.off_codes[c]);
      mat.off_scales[c] = opaque(mat.off_scales[c]);
      mat.n_entries[c] = opaque(mat.n_entries[c]);
    }
    WinCounts wc;
    wc.own[0] = own.x;
    wc.own[1] = own.y;
    wc.own[2] = own.z;
    wc.own[3] = own.w;
    const uint32_t es[4] = {erow.x, erow.y, erow.z, erow.w};
    uint32_t o = 0;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      wc.before[c] = 0u;
      start[c] = es[c];
      n[c] = clamp_run(mat, c, start[c], wc.own[c]);
      seg[c] = inv + 2u * o;
      o += wc.own[c];
    }
    if (role == 0) {
      load_batch<0, MT>(A0, mat, start[0], n[0], 0, lane);
      load_batch<3, MT>(A3, mat, start[3], n[3], 0, lane);
      build_index(wr, u, 0, u.W, R, wc, inv, lane);
    } else {
      load_batch<1, MT>(A1, mat, start[1], n[1], 0, lane);
      load_batch<2, MT>(A2, mat, start[2], n[2], 0, lane);
      if constexpr (MT == 1)
        store_x1(u.cols, xr, wn, lane);
      else
        store_xm<MT>(a, u.cols, xrm, wn, lane);
    }
  }
  __syncthreads();  // the index and x of every unit are in LDS
  if (active) {
    if (role == 0) {
      run_class<0, MT>(mat, A0, start[0], n[0], seg[0], wn, lane);
      run_class<3, MT>(mat, A3, start[3], n[3], seg[3], wn, lane);
    } else {
      run_class<1, MT>(mat, A1, start[1], n[1], seg[1], wn, lane);
      run_class<2, MT>(mat, A2, start[2], n[2], seg[2], wn, lane);
    }
  }
  __syncthreads();  // every partial product is in LDS
  if (active && role == 0) reduce_window<MT>(wn, R, u.cols, u.rows, ysum, lane);
  __syncthreads();
  const int rows = min(R, mat.N - t * R);
  for (int slot = threadIdx.x; slot < MT * R; slot += NW * 64) {
    const int m = slot >> mat.logR, r = slot & (R - 1);
    if (m < a.M && r < rows) {
      float tot = 0.0f;
#pragma unroll
      for (int p2 = 0; p2 < NP; ++p2) tot += lds_f32(lds0 + 4u * (uint32_t)(p2 * MT * R + slot));
      if constexpr (MT == 1)
        store_row(a, (size_t)t * R + r, tot);
      else
        store_y(a.y, m * a.ldy + (size_t)t * R + r, tot, a.yf16);
    }
  }
}

// ---------------------------------------------------------------------------
// Several activation rows (3 <= M <= 16): matrix cores.
//
// Y[m][n] = sum_k w_hat[n][k] X[m][k] as 16 x 16 x 16 fp16 MFMA products
// D[m][r] = sum_k X[m][k] q_r[k] over the 16 entries r of one group column
// and 16 consecutive rows (a "block"), whatever their widths:
//   * lane l works for weight row r = l % 16 and, over the four products kb,
//     for group positions 16 (l/16) .. + 15 (product kb takes 16 (l/16) + 4 kb
//     .. + 3: the k order inside a product is free as long as A and B agree);
//   * A: activations X[l % 16][64 col + 16 (l/16) ..] (two 16-byte loads);
//   * B: the levels q of row r's entry, made exactly in fp16: a code field ORed
//     into the mantissa of 1024.0 reads as 1024 + u, and packed fp16 adds give
//     q.  Each lane decodes its own entry's width with per-lane field
//     positions, masks and offsets, so every lane runs the same code;
//   * D: lane l holds D[4 (l/16) + j][l % 16], j = 0..3, so each lane adds
//     s * D for its weight row and four activation rows to registers over the
//     slice's columns, in column order (results are bitwise repeatable).
// A position's entry comes from a per-slice map position -> (class, rank in
// the slice's class run) built from the width map.
// ---------------------------------------------------------------------------
typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef float float4_t __attribute__((ext_vector_type(4)));

constexpr int kMmRows = 16;
constexpr int kMmMaxCols = 32;  // group columns of a slice

struct MmArgs {
  DevMatrix m;
  const uint16_t* x;  // fp16 bits, row m at x + m*ldx
  void* y;            // row m at y + m*ldy elements (float, or fp16 bits when yf16)
  int64_t ldx, ldy;
  int32_t M;          // rows of X (3..16)
  int32_t S;          // slices per unit
  int32_t yf16;       // 1: y holds fp16
};

// Bytes of one wave's LDS region: row sums (16 x R floats), the per-class
// table of the slice (five rows of eight words), and the position -> entry
// map (uint16 per position of the widest slice).
constexpr int kMmTableBytes = 5 * 32;
__host__ __device__ inline int mm_wave_bytes(int R, int cols) {
  return kMmRows * R * 4 + kMmTableBytes + align16(((cols * R + 63) / 64) * 64 * 2);
}

// The table a lane reads for its block's entry, row c of width class c (row
// 4: class 0 for lanes with odd h, whose 1-bit fields sit 8 bits higher):
//   word 0..3  code section offset, scale section offset, slice run start,
//              last entry of the class section (addresses of the entry);
//   word 4     field mask of one pair (two codes, one per half-word): 1 bit
//              codes are read from the word rotated right by 31 (even h:
//              fields 0..7 move up one bit) or by 7 (odd h: fields 8..15 move
//              down seven), so a field shifted by its offset lands at bit 1 of
//              each half, and no field crosses the word's ends;
//   word 5     -(1024 + offset) in both fp16 halves: a masked field ORed into
//              1024.0 reads as 1024 + u (1024 + 2u for 1 bit), and one
//              packed add makes the level q exactly (1025 for 1 bit, 1024 +
//              2^(b-1) otherwise: integers below 2048, exact in fp16);
//   word 6     the field's bit offset (in the rotated word) for products
//              kb = 0..3, one per byte;
//   word 7     the pair's second field offset b | (3 + c) << 8 (log2 of the
//              entry's bytes) | c << 16 | rotation << 24.
// Row `row` of the table (lane 0 of the wave writes all five once per slice;
// the values are wave-uniform): code and scale section offsets, the slice's
// run start and the class section's last entry.
template <int row>
__device__ __forceinline__ void write_mm_row(uint32_t tab, uint32_t offc, uint32_t offs, uint32_t start,
                                             uint32_t lim) {
  constexpr uint32_t c = row == 4 ? 0u : (uint32_t)row;
  constexpr uint32_t kMask[4] = {0x00020002u, 0x00030003u, 0x000F000Fu, 0x00FF00FFu};
  constexpr uint32_t kSub[4] = {0xE401E401u, 0xE402E402u, 0xE408E408u, 0xE480E480u};
  constexpr uint32_t kShift[4] = {0x06040200u, 0x0C080400u, 0x08000800u, 0u};
  constexpr uint32_t rot = row == 4 ? 7u : row == 0 ? 31u : 0u;
  lds_store_u32x4(tab + 32u * row, u32x4{offc, offs, start, lim});
  lds_store_u32x4(tab + 32u * row + 16u,
                  u32x4{kMask[c], kSub[c], kShift[c], (1u << c) | ((3u + c) << 8) | (c << 16) | (rot << 24)});
}

// One block in registers for this lane: its entry's 16 code bytes that hold
// the lane's 16 levels, the class table's decoding words, the fp16 scale bits
// (zero-extended), and 16 activations of row l % 16.  A lane of a padding row
// (past the matrix's last row) decodes a clamped in-range entry: its product
// column is that row's alone and is never added to a row sum, so no value
// loaded for it needs a select (which would wait for the load).
struct MmBlock {
  u32x4 w;
  u32x4 k;   // table words 4..7 of the entry's class
  uint32_t s;
  u32x4 a0, a1;
};

// Block f of the row group: column f / RB, row block rg*RB + f % RB.  The
// lane's levels 16h .. 16h + 15 (h = lane / 16) are pairs 8h .. 8h + 7, whose
// codes start at byte (2h << c) & ~3 of the entry.  Loads are unconditional
// (clamped), so the next block stays in flight.  X comes through a buffer
// resource (xr) covering the M rows.
template <int RB>
__device__ __forceinline__ void load_mm_block(MmBlock& bk, __amdgpu_buffer_rsrc_t xr, int64_t ldx, int M,
                                              const DevMatrix& mat, uint32_t fwd, uint32_t tab, int f, int rg,
                                              int rows, int j0, uint32_t lane) {
  const int R = mat.R;
  const uint32_t e = lane & 15u, h = lane >> 4;
  const int col = f / RB;
  const int row = (rg * RB + f % RB) * 16 + (int)e;
  const uint32_t v = (uint32_t)lds_u16(fwd + 2u * (uint32_t)(col * R + row));
  const bool real = row < rows;
  const uint32_t c = real ? v >> 14 : 0u;
  const uint32_t trow = (c == 0u && (h & 1u)) ? 4u : c;
  const u32x4 t0 = lds_u32x4(tab + 32u * trow);
  bk.k = lds_u32x4(tab + 32u * trow + 16u);
  const uint32_t g = min(t0.z + (real ? (v & 0x3FFFu) : 0u), t0.w);
  bk.w = ld<u32x4>(mat.blob, t0.x + (g << (3 + c)) + (((2u * h) << c) & ~3u));
  bk.s = (uint32_t)ld<uint16_t>(mat.blob, t0.y + 2u * g);
  const int m = min((int)e, M - 1);
  const uint32_t xo = 2u * (uint32_t)((int64_t)m * ldx + (int64_t)(j0 + col) * 64 + 16 * (int)h);
  bk.a0 = __builtin_amdgcn_raw_buffer_load_b128(xr, (int)xo, 0, 0);
  bk.a1 = __builtin_amdgcn_raw_buffer_load_b128(xr, (int)xo + 16, 0, 0);
}

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));

// s * D of one block, two 16 x 16 x 32 products (weights 16h .. 16h + 7 and
// 16h + 8 .. 16h + 15 of the lane's entry against the same activations).
// For kb = 0..3 the lane's pairs 8h + 2kb, + 1 are fields f, f + 1 of word
// wi of its 16 code bytes:
//   1 bit: wi = 0, f = 8 (h & 1) + 2kb;  2 bits: wi = 0, f = 2kb;
//   4 bits: wi = kb / 2, f = 2 (kb & 1); 8 bits: wi = kb, f = 0.
__device__ __forceinline__ float4_t mm_products(const MmBlock& bk) {
  const uint32_t c = (bk.k.w >> 16) & 0xFFu, B = bk.k.w & 0xFFu;
  const uint32_t mask = bk.k.x, sub = bk.k.y, shifts = bk.k.z;
  const uint32_t src0 = __builtin_amdgcn_alignbit(bk.w.x, bk.w.x, bk.k.w >> 24);
  const uint32_t src1 = c == 3u ? bk.w.y : src0;
  const uint32_t src2 = c == 3u ? bk.w.z : c == 2u ? bk.w.y : src0;
  const uint32_t src3 = c == 3u ? bk.w.w : c == 2u ? bk.w.y : src0;
  const uint32_t word[4] = {src0, src1, src2, src3};
  uint32_t q[8];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    const uint32_t sh = (shifts >> (8 * kb)) & 0xFFu;
    const uint32_t v0 = ((word[kb] >> sh) & mask) | 0x64006400u;  // 1024 + u (1024 + 2u for 1 bit)
    const uint32_t v1 = ((word[kb] >> (sh + B)) & mask) | 0x64006400u;
    q[2 * kb] = __builtin_bit_cast(uint32_t, as_h2(v0) + as_h2(sub));
    q[2 * kb + 1] = __builtin_bit_cast(uint32_t, as_h2(v1) + as_h2(sub));
  }
  const half8_t b0 = __builtin_bit_cast(half8_t, u32x4{q[0], q[1], q[2], q[3]});
  const half8_t b1 = __builtin_bit_cast(half8_t, u32x4{q[4], q[5], q[6], q[7]});
  float4_t d = {0.0f, 0.0f, 0.0f, 0.0f};
  d = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8_t, bk.a0), b0, d, 0, 0, 0);
  d = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8_t, bk.a1), b1, d, 0, 0, 0);
  const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)bk.s);
  return d * s;
}

// Marks a block's registers as read here: every buffer's load is consumed on
// every path, so no register with a load in flight is ever reused for
// something else (which would make the compiler wait for all loads).
__device__ __forceinline__ void mm_done(const MmBlock& bk) {
  __asm__ __volatile__("" ::"v"(bk.w), "v"(bk.s), "v"(bk.a0), "v"(bk.a1), "v"(bk.k));
}

// As for the one-row kernel, the values the first loads depend on come as
// preloaded leading arguments (geo packs R, C, log2 R and S the same way),
// the unit table is read beside the width map rather than after it, and the
// argument block is read only once those loads are issued.
template <int NW, int RB>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(4))) void vbq_mm_kernel(const uint8_t* __restrict__ blob, uint32_t off_wmap,
                                                         uint32_t tile_words, uint32_t chunk_words, uint32_t wmap_words,
                                                         int32_t G, int32_t N, uint32_t geo, int32_t U, MmArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  DevMatrix mat = a.m;
  mat.blob = blob;
  mat.off_wmap = off_wmap;
  mat.tile_words = tile_words;
  mat.chunk_words = chunk_words;
  mat.wmap_words = wmap_words;
  mat.G = G;
  mat.N = N;
  mat.U = U;
  mat.R = (int)(geo & 0x1FF);
  mat.C = (int)((geo >> 9) & 0xFF);
  mat.logR = (int)((geo >> 17) & 0xF);
  const int R = mat.R, S = (int)((geo >> 21) & 0x3FF);
  const bool setup_prio = (geo >> 31) != 0u;  // raised issue priority for each item's set-up
  const uint32_t lds0 = (uint32_t)(size_t)(__attribute__((address_space(3))) uint8_t*)smem;
  const int wave = wave_id();
  const int t = blockIdx.x;  // one row tile per workgroup
  const int cmax = max_slice_cols(R, mat.C, S);
  const int wbytes = mm_wave_bytes(R, cmax);
  const uint32_t ysum = lds0 + (uint32_t)(wave * wbytes);
  const uint32_t tab = ysum + (uint32_t)(kMmRows * R * 4);
  const uint32_t fwd = tab + (uint32_t)kMmTableBytes;
  const int rows = min(R, mat.N - t * R);
  {
    const uint32_t lane = lane_id_here();
    for (int i = (int)lane; i < kMmRows * R; i += 64) lds_store_f32(ysum + 4u * i, 0.0f);
  }
  for (int item = wave; item < mat.U * S; item += NW) {
    const uint32_t lane = lane_id_here();
    const uint32_t h = lane >> 4;
    const int k = item / S, sl = item - k * S;
    const UnitInfo u = load_unit(mat, t, k);
    const int unit = t * mat.U + k;
    int cb, ce;
    slice_cols(u.cols, R, sl, S, cb, ce);
    if (cb >= ce) continue;  // wave-uniform: an empty slice
    if (setup_prio) __builtin_amdgcn_s_setprio(1);
    const int wb = (cb * R) >> 6, we = (ce * R + 63) >> 6;
    const WmapRegs wr = load_wmap(mat, u, we, lane);
    const u32x16 rows2 = unit_rows_vec(mat, unit);  // beside the width map, not after it
    const uint32_t es[4] = {rows2.s0, rows2.s1, rows2.s2, rows2.s3};
    // values from the kernel-argument block only after the loads above are
    // issued (the compiler would otherwise hoist them and wait for the block)
    lds_phase();
    const uint16_t* xp = (const uint16_t*)opaque64((uint64_t)a.x);
    const int64_t ldx = (int64_t)opaque64((uint64_t)a.ldx);
    const int M = (int)opaque((uint32_t)a.M);
    // X rows 0 .. M-1 (fp16, stride ldx): the bytes up to the end of row M-1
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)xp, 0, (int)(2 * ((int64_t)(M - 1) * ldx + mat.K)), 0x00020000);
    const WinCounts wc = window_counts(wr, u, wb, we, R, lane);
#define VBQ_MM_ROW(row, c)                                                                          \
  write_mm_row<row>(tab, opaque(mat.off_codes[c]), opaque(mat.off_scales[c]),                       \
                    uniform((int)(es[c] + wc.before[c])), uniform((int)(max(opaque(mat.n_entries[c]), 1u) - 1u)))
    if (lane == 0) {
      VBQ_MM_ROW(0, 0);
      VBQ_MM_ROW(1, 1);
      VBQ_MM_ROW(2, 2);
      VBQ_MM_ROW(3, 3);
      VBQ_MM_ROW(4, 0);
    }
#undef VBQ_MM_ROW
    build_index<true>(wr, u, wb, we, R, wc, fwd, lane);
    lds_phase();
    if (setup_prio) __builtin_amdgcn_s_setprio(0);
    const int j0 = u.j0 + cb;
    const int nf = (ce - cb) * RB;  // blocks per row group
    const int last = nf - 1;
    for (int rg = 0; rg < R / (16 * RB); ++rg) {
      float4_t acc[RB];
#pragma unroll
      for (int i = 0; i < RB; ++i) acc[i] = float4_t{0.0f, 0.0f, 0.0f, 0.0f};
      // Two blocks in flight (the next one loads while one is multiplied):
      // with four, every wave's chain of index lookups and loads got longer
      // (1.46B-class step at M = 4: 1415 against 1262 us).  With more than
      // four rows of X, tiles of one or four row blocks take one block at a
      // time (their blocks read more X; at M = 16 the step took 1551 against
      // 1603 us, at M = 4 it would take 1281 against 1264).  Block f adds
      // into acc[f % RB] (the ring slot) either way.
      MmBlock B0, B1;
      if (RB != 2 && M > 4) {  // wave-uniform
        for (int f = 0; f < nf; ++f) {
          load_mm_block<RB>(B0, xr, ldx, M, mat, fwd, tab, f, rg, rows, j0, lane);
          acc[f % RB] += mm_products(B0);
          mm_done(B0);
        }
      } else {
      load_mm_block<RB>(B0, xr, ldx, M, mat, fwd, tab, 0, rg, rows, j0, lane);
      for (int f = 0; f < nf; f += 4) {
        load_mm_block<RB>(B1, xr, ldx, M, mat, fwd, tab, min(f + 1, last), rg, rows, j0, lane);
        acc[0 % RB] += mm_products(B0);
        mm_done(B0);
        load_mm_block<RB>(B0, xr, ldx, M, mat, fwd, tab, min(f + 2, last), rg, rows, j0, lane);
        if (f + 1 < nf) acc[1 % RB] += mm_products(B1);
        mm_done(B1);
        load_mm_block<RB>(B1, xr, ldx, M, mat, fwd, tab, min(f + 3, last), rg, rows, j0, lane);
        if (f + 2 < nf) acc[2 % RB] += mm_products(B0);
        mm_done(B0);
        load_mm_block<RB>(B0, xr, ldx, M, mat, fwd, tab, min(f + 4, last), rg, rows, j0, lane);
        if (f + 3 < nf) acc[3 % RB] += mm_products(B1);
        mm_done(B1);
      }
      mm_done(B0);
      }
      // this wave's share of the row sums (several items add up in order)
#pragma unroll
      for (int i = 0; i < RB; ++i) {
        const int row = (rg * RB + i) * 16 + (int)(lane & 15u);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int m = 4 * (int)h + j;
          if (m < M && row < rows) {
            const uint32_t ya = ysum + 4u * (uint32_t)(m * R + row);
            lds_store_f32(ya, lds_f32(ya) + acc[i][j]);
          }
        }
      }
    }
    lds_phase();
  }
  __syncthreads();
  for (int slot = threadIdx.x; slot < kMmRows * R; slot += NW * 64) {
    const int m = slot / R, r = slot - m * R;
    if (m < a.M && r < rows) {
      float tot = 0.0f;
#pragma unroll
      for (int w2 = 0; w2 < NW; ++w2) tot += lds_f32(lds0 + (uint32_t)(w2 * wbytes) + 4u * (uint32_t)slot);
      store_y(a.y, m * a.ldy + (size_t)t * R + r, tot, a.yf16);
    }
  }
}

// w_hat = s*q written densely (checking aid, not a hot path): four waves per
// tile, each indexing slice `wave` of every unit (one window) and writing its
// entries, one lane per entry.
constexpr int kDequantWaves = 4;

__global__ __launch_bounds__(kDequantWaves * 64) void vbq_dequant_kernel(DevMatrix mat, float* W, int region_bytes) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const uint32_t lane = lane_id();
  const int wave = wave_id();
  const int t = blockIdx.x;
  const int R = mat.R;
  const uint32_t inv = (uint32_t)(size_t)(__attribute__((address_space(3))) uint8_t*)smem + (uint32_t)(wave * region_bytes);
  for (int k = 0; k < mat.U; ++k) {
    const UnitInfo u = load_unit(mat, t, k);
    const int unit = t * mat.U + k;
    int cb, ce;
    slice_cols(u.cols, R, wave, kDequantWaves, cb, ce);
    if (cb >= ce) continue;
    const int wb = (cb * R) >> 6, we = (ce * R + 63) >> 6;
    const WmapRegs wr = load_wmap(mat, u, we, lane);
    const WinCounts wc = window_counts(wr, u, wb, we, R, lane);
    build_index(wr, u, wb, we, R, wc, inv, lane);
    lds_phase();
    uint32_t seg = inv;
    for (int c = 0; c < 4; ++c) {
      const int B = 1 << c, NWc = 2 * B, per = 16 / B;
      const uint32_t mask = (1u << B) - 1;
      const uint32_t start = class_start(mat, unit, c) + wc.before[c];
      const int n = clamp_run(mat, c, start, wc.own[c]);
      for (int e = (int)lane; e < n; e += 64) {
        const int p = lds_u16(seg + 2u * (uint32_t)e) + wb * 64;  // unit position
        const int jl = p >> mat.logR, r = p & (R - 1);
        const size_t g = (size_t)start + e;
        const uint32_t* wv = (const uint32_t*)(mat.blob + mat.off_codes[c]) + g * NWc;
        const float s = (float)__builtin_bit_cast(_Float16, ld<uint16_t>(mat.blob, mat.off_scales[c] + 2u * (uint32_t)g));
        float* dst = W + ((size_t)t * R + r) * mat.K + (size_t)(u.j0 + jl) * 64;
        for (int i = 0; i < 32; ++i) {
          const uint32_t word = wv[i / per];
          const int f = i % per;
          const int u0 = (int)((word >> (f * B)) & mask), u1 = (int)((word >> (16 + f * B)) & mask);
          const int q0 = c == 0 ? 2 * u0 - 1 : u0 - (1 << (B - 1));
          const int q1 = c == 0 ? 2 * u1 - 1 : u1 - (1 << (B - 1));
          dst[2 * i] = s * (float)q0;
          dst[2 * i + 1] = s * (float)q1;
        }
      }
      seg += 2u * wc.own[c];
    }
    lds_phase();
  }
}

thread_local hipError_t g_last_hip_error = hipSuccess;

vbq_status hip_status(hipError_t e) {
  if (e == hipSuccess) return VBQ_OK;
  g_last_hip_error = e;
  return VBQ_ERR_HIP;
}

vbq_status make_dev_matrix(const vbq_desc* d, const void* blob, DevMatrix* m) {
  if (!d || !blob) return VBQ_ERR_NULL;
  vbq_status st = vbq_desc_check(d);
  if (st != VBQ_OK) return st;
  if ((uintptr_t)blob % 256 != 0) return VBQ_ERR_BUFFER;
  if (d->total_bytes >= (1ull << 32)) return VBQ_ERR_UNSUPPORTED;  // 32-bit section offsets
  // the kernels address the unit table at offset 0 (the layout's first section)
  if (d->section_off[VBQ_SEC_UNITS] != 0) return VBQ_ERR_DESC;
  if (d->flags & ~(uint32_t)VBQ_CALL_FLAGS) return VBQ_ERR_UNSUPPORTED;
  m->blob = (const uint8_t*)blob;
  m->off_units = 0;
  m->off_wmap = (uint32_t)d->section_off[VBQ_SEC_WMAP];
  for (int c = 0; c < 4; ++c) {
    m->n_entries[c] = (uint32_t)d->n_entries[c];
    // loads of an empty class are clamped to the unit table's first bytes
    m->off_codes[c] = m->n_entries[c] ? (uint32_t)d->section_off[VBQ_SEC_CODES0 + c] : m->off_units;
    m->off_scales[c] = m->n_entries[c] ? (uint32_t)d->section_off[VBQ_SEC_SCALES0 + c] : m->off_units;
  }
  m->wmap_words = (uint32_t)(d->section_len[VBQ_SEC_WMAP] / 8);
  if (m->wmap_words == 0) return VBQ_ERR_DESC;
  {
    const int64_t G = d->K / 64, C = d->chunk_groups, R = d->tile_rows, U = d->n_chunks;
    const int64_t wf = (C * R + 63) / 64, wl = ((G - (U - 1) * C) * R + 63) / 64;
    m->chunk_words = (uint32_t)wf;
    m->tile_words = (uint32_t)(2 * ((U - 1) * wf + wl));
    if ((uint64_t)m->tile_words * (uint64_t)d->n_tiles != m->wmap_words) return VBQ_ERR_DESC;
  }
  m->N = (int32_t)d->N;
  m->K = (int32_t)d->K;
  m->G = (int32_t)(d->K / 64);
  m->R = d->tile_rows;
  m->C = d->chunk_groups;
  m->T = (int32_t)d->n_tiles;
  m->U = (int32_t)d->n_chunks;
  int lr = 0;
  while ((1 << lr) < m->R) ++lr;
  m->logR = lr;
  return VBQ_OK;
}

constexpr int kLdsLimit = 160 * 1024;
constexpr int kMinWaves = 4;

// Launch shape of the fused product for MT activation rows.
struct MvShape {
  int NW;  // waves per workgroup (4, 8 or 16)
  int S;   // slices per unit
  int SW;  // window columns
  int lds; // dynamic LDS bytes
};

// Slices per unit: enough for four per tile, and for one activation row
// narrow enough for the window to be the whole slice (at most 32 columns of
// x held in registers).  Waves per workgroup: one per (unit, slice) item, as
// a power of two from 4 to 16 (8 for several rows), so that a wave's items
// (a chain of dependent loads each) run side by side rather than in turn.
// Window: the whole slice if it fits the LDS budget (64 KB, else the 160 KB
// of a CU), else the largest multiple of the columns per width-map word
// that does.
bool choose_shape(const DevMatrix& m, int MT, MvShape* sh) {
  int S = (kMinWaves + m.U - 1) / m.U;
  if (MT == 1)
    while (max_slice_cols(m.R, m.C, S) > kXRegs * 8) ++S;
  const int max_nw = MT == 1 ? 16 : 8;  // several rows need more than 128 VGPRs: 2 waves per SIMD
  int NW = kMinWaves;
  while (NW < max_nw && NW < m.U * S) NW *= 2;
  const int cw = cols_per_word(m.R);
  const int full = max_slice_cols(m.R, m.C, S);
  int SW = 0;
  if (MT == 1) {
    if (mv_lds_bytes(m.R, full, 1, NW) <= kLdsLimit) SW = full;
  } else {
    for (int limit : {64 * 1024, kLdsLimit}) {
      if (mv_lds_bytes(m.R, full, MT, NW) <= limit) {
        SW = full;
        break;
      }
      for (int sw = (full / cw) * cw; sw >= cw && !SW; sw -= cw)
        if (mv_lds_bytes(m.R, sw, MT, NW) <= limit) SW = sw;
      if (SW) break;
    }
  }
  if (SW <= 0) return false;
  sh->NW = NW;
  sh->S = S;
  sh->SW = SW;
  sh->lds = mv_lds_bytes(m.R, SW, MT, NW);
  return true;
}

// Raises a kernel's dynamic LDS limit once per device.
vbq_status allow_big_lds(const void* kernel, std::atomic<uint64_t>& done) {
  int dev = 0;
  vbq_status st = hip_status(hipGetDevice(&dev));
  if (st != VBQ_OK) return st;
  const uint64_t bit = 1ull << (dev & 63);
  if (done.load(std::memory_order_acquire) & bit) return VBQ_OK;
  st = hip_status(hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, kLdsLimit));
  if (st == VBQ_OK) done.fetch_or(bit, std::memory_order_release);
  return st;
}

template <int MT, int NW, int UNI = -1>
vbq_status launch_mv_nw(const MvArgs& a, int lds, hipStream_t s) {
  const void* kernel = (const void*)vbq_mv_kernel<MT, NW, UNI>;
  if (lds > 64 * 1024) {  // beyond the default dynamic LDS limit
    static std::atomic<uint64_t> done{0};
    vbq_status st = allow_big_lds(kernel, done);
    if (st != VBQ_OK) return st;
  }
  MvArgs args = a;
  const uint16_t* x = a.x;
  const uint8_t* blob = a.m.blob;
  uint32_t off_wmap = a.m.off_wmap, tile_words = a.m.tile_words, chunk_words = a.m.chunk_words;
  if constexpr (UNI >= 0) {  // (the kernel reads them as such)
    off_wmap = a.m.off_codes[UNI];
    tile_words = a.m.off_scales[UNI];
    chunk_words = a.m.n_entries[UNI];
  }
  uint32_t wmap_words = a.m.wmap_words;
  int32_t G = a.m.G, N = a.m.N, U = a.m.U;
  uint32_t geo = (uint32_t)a.m.R | ((uint32_t)a.m.C << 9) | ((uint32_t)a.m.logR << 17) | ((uint32_t)a.S << 21);
  uint32_t sw_m = (uint32_t)a.SW | ((uint32_t)a.M << 16);
  void* kargs[] = {&x, &blob, &off_wmap, &tile_words, &chunk_words, &wmap_words, &G, &N, &geo, &U, &sw_m, &args};
  return hip_status(hipLaunchKernel(kernel, dim3((unsigned)a.m.T), dim3(NW * 64), kargs, (size_t)lds, s));
}

// Wave pairs: one or two rows, mixed widths, whole units of at most 32
// columns, at most 8 units per tile (4 for two rows), and a grid small enough
// that one wave per unit would leave the SIMDs with at most two waves each.
constexpr int kPairMaxUnits = 2048;

template <int NW, int MT>
vbq_status launch_pair_nw(const MvArgs& a, int lds, hipStream_t s) {
  const void* kernel = (const void*)vbq_mv_pair_kernel<NW, MT>;
  if (lds > 64 * 1024) {
    static std::atomic<uint64_t> done{0};
    vbq_status st = allow_big_lds(kernel, done);
    if (st != VBQ_OK) return st;
  }
  MvArgs args = a;
  const uint16_t* x = a.x;
  const uint8_t* blob = a.m.blob;
  uint32_t off_wmap = a.m.off_wmap, tile_words = a.m.tile_words, chunk_words = a.m.chunk_words;
  uint32_t wmap_words = a.m.wmap_words;
  int32_t G = a.m.G, N = a.m.N, U = a.m.U;
  uint32_t geo = (uint32_t)a.m.R | ((uint32_t)a.m.C << 9) | ((uint32_t)a.m.logR << 17) | (1u << 21);
  uint32_t sw_m = (uint32_t)a.SW | ((uint32_t)a.M << 16);
  void* kargs[] = {&x, &blob, &off_wmap, &tile_words, &chunk_words, &wmap_words, &G, &N, &geo, &U, &sw_m, &args};
  return hip_status(hipLaunchKernel(kernel, dim3((unsigned)a.m.T), dim3(NW * 64), kargs, (size_t)lds, s));
}

// Waves per workgroup of the pair kernel for MT (1 or 2) activation rows, or
// 0 when the matrix does not qualify.
int pair_waves(const DevMatrix& m, int MT) {
  int classes = 0;
  for (int c = 0; c < 4; ++c) classes += m.n_entries[c] ? 1 : 0;
  if (classes < 2 || m.U < 2 || m.U > 8 || m.C > kXRegs * 8) return 0;
  if ((int64_t)m.T * m.U > kPairMaxUnits) return 0;
  // two rows fit the registers of 8 waves per workgroup (2 per SIMD), not of 16
  if (MT > 1 && m.U > 4) return 0;
  const int NW = m.U <= 4 ? 8 : 16;
  const int lds = (NW / 2) * (MT * m.R * 4 + wave_plan(m.R, m.C, MT).bytes);
  return lds > kLdsLimit ? 0 : NW;
}

// Launches the pair kernel for MT (1 or 2) activation rows when the matrix
// qualifies; *used says whether it did.
template <int MT>
vbq_status try_launch_pair(const DevMatrix& m, const void* x, int64_t ldx, void* y, int64_t ldy, bool yf16,
                           const int32_t* rows, int64_t ylen, hipStream_t s, bool* used) {
  *used = false;
  const int NW = pair_waves(m, MT);
  if (NW == 0) return VBQ_OK;
  const int lds = (NW / 2) * (MT * m.R * 4 + wave_plan(m.R, m.C, MT).bytes);
  MvArgs a;
  a.m = m;
  a.x = (const uint16_t*)x;
  a.y = y;
  a.ldx = ldx;
  a.ldy = ldy;
  a.M = MT;
  a.S = 1;
  a.SW = m.C;
  a.yf16 = yf16 ? 1 : 0;
  a.rows = MT == 1 ? rows : nullptr;
  a.ylen = ylen;
  *used = true;
  if constexpr (MT == 1)
    if (NW == 16) return launch_pair_nw<16, 1>(a, lds, s);
  return launch_pair_nw<8, MT>(a, lds, s);
}

// flags: the descriptor's call options (VBQ_Y_F16, VBQ_ONE_WAVE_PER_UNIT).
template <int MT>
vbq_status launch_mv(const DevMatrix& m, uint32_t flags, const void* x, int64_t ldx, int M, void* y, int64_t ldy,
                     hipStream_t s, const int32_t* rows = nullptr, int64_t ylen = 0) {
  const bool yf16 = (flags & VBQ_Y_F16) != 0;
  if constexpr (MT <= 2) {
    if (!(flags & VBQ_ONE_WAVE_PER_UNIT)) {
      bool used = false;
      const vbq_status st = try_launch_pair<MT>(m, x, ldx, y, ldy, yf16, rows, ylen, s, &used);
      if (used) return st;
    }
  }
  MvShape sh;
  if (!choose_shape(m, MT, &sh)) return VBQ_ERR_UNSUPPORTED;
  MvArgs a;
  a.m = m;
  a.x = (const uint16_t*)x;
  a.y = y;
  a.ldx = ldx;
  a.ldy = ldy;
  a.M = M;
  a.S = sh.S;
  a.SW = sh.SW;
  a.yf16 = yf16 ? 1 : 0;
  a.rows = MT == 1 ? rows : nullptr;
  a.ylen = ylen;
  if constexpr (MT == 1) {
    // a matrix of one width class (a "recipe" matrix) takes the uniform kernel
    int uni = -1, classes = 0;
    for (int c = 0; c < 4; ++c)
      if (m.n_entries[c]) {
        uni = c;
        ++classes;
      }
    if (classes == 1) {
      // no position index; the 1-bit kernel holds one group column's lookup
      // tables per wave
      sh.lds = mv_lds_bytes(m.R, sh.SW, 1, sh.NW, uni == 0 ? kLutBytes : 0, false);
      if (sh.lds > kLdsLimit) return VBQ_ERR_UNSUPPORTED;
      switch (uni * 3 + (sh.NW == 4 ? 0 : sh.NW == 8 ? 1 : 2)) {
        case 0: return launch_mv_nw<1, 4, 0>(a, sh.lds, s);
        case 1: return launch_mv_nw<1, 8, 0>(a, sh.lds, s);
        case 2: return launch_mv_nw<1, 16, 0>(a, sh.lds, s);
        case 3: return launch_mv_nw<1, 4, 1>(a, sh.lds, s);
        case 4: return launch_mv_nw<1, 8, 1>(a, sh.lds, s);
        case 5: return launch_mv_nw<1, 16, 1>(a, sh.lds, s);
        case 6: return launch_mv_nw<1, 4, 2>(a, sh.lds, s);
        case 7: return launch_mv_nw<1, 8, 2>(a, sh.lds, s);
        case 8: return launch_mv_nw<1, 16, 2>(a, sh.lds, s);
        case 9: return launch_mv_nw<1, 4, 3>(a, sh.lds, s);
        case 10: return launch_mv_nw<1, 8, 3>(a, sh.lds, s);
        default: return launch_mv_nw<1, 16, 3>(a, sh.lds, s);
      }
    }
  }
  if (sh.NW == 4) return launch_mv_nw<MT, 4>(a, sh.lds, s);
  if constexpr (MT == 1) {
    if (sh.NW == 16) return launch_mv_nw<MT, 16>(a, sh.lds, s);
  }
  return launch_mv_nw<MT, 8>(a, sh.lds, s);
}

// Several rows on matrix cores: same item split as the one-row path (slices
// of at most 32 columns, at least four items per tile).
template <int NW, int RB>
vbq_status launch_mm_nw(const MmArgs& a, int lds, hipStream_t s) {
  const void* kernel = (const void*)vbq_mm_kernel<NW, RB>;
  if (lds > 64 * 1024) {
    static std::atomic<uint64_t> done{0};
    vbq_status st = allow_big_lds(kernel, done);
    if (st != VBQ_OK) return st;
  }
  MmArgs args = a;
  const uint8_t* blob = a.m.blob;
  uint32_t off_wmap = a.m.off_wmap, tile_words = a.m.tile_words, chunk_words = a.m.chunk_words;
  uint32_t wmap_words = a.m.wmap_words;
  int32_t G = a.m.G, N = a.m.N, U = a.m.U;
  // bit 31: each item's set-up (width map, class runs, index) at a raised issue
  // priority, for up to eight rows (1.46B-class step: M = 4 1271 -> 1260 us, M = 8
  // 1343 -> 1326 us; at M = 16 it was slower, 1548 -> 1555 us)
  uint32_t geo = (uint32_t)a.m.R | ((uint32_t)a.m.C << 9) | ((uint32_t)a.m.logR << 17) | ((uint32_t)a.S << 21) |
                 (a.M <= 8 ? 1u << 31 : 0u);
  void* kargs[] = {&blob, &off_wmap, &tile_words, &chunk_words, &wmap_words, &G, &N, &geo, &U, &args};
  return hip_status(hipLaunchKernel(kernel, dim3((unsigned)a.m.T), dim3(NW * 64), kargs, (size_t)lds, s));
}

template <int RB>
vbq_status launch_mm_rb(const MmArgs& a, int NW, int lds, hipStream_t s) {
  if (NW == 4) return launch_mm_nw<4, RB>(a, lds, s);
  if (NW == 8) return launch_mm_nw<8, RB>(a, lds, s);
  return launch_mm_nw<16, RB>(a, lds, s);
}

// Launch shape of the matrix-core kernel: waves per workgroup, slices per
// unit, LDS bytes.  Each wave walks its blocks one after the other, so small
// matrices split their tiles over more waves, as long as the whole grid fits
// the GPU at once (about 20 waves per CU at this kernel's register use).
bool mm_shape(const DevMatrix& m, int* NWo, int* So, int* ldso) {
  int NWt = kMinWaves;
  while (NWt < 16 && (int64_t)m.T * NWt * 2 <= 256 * 20) NWt *= 2;
  int S = (NWt + m.U - 1) / m.U;
  while (max_slice_cols(m.R, m.C, S) > kMmMaxCols) ++S;
  const int wbytes = mm_wave_bytes(m.R, max_slice_cols(m.R, m.C, S));
  int NW = kMinWaves;  // (fewer waves than items is fine: items are dealt in turn)
  while (NW < 16 && NW < m.U * S && 2 * NW * wbytes <= kLdsLimit) NW *= 2;
  *NWo = NW;
  *So = S;
  *ldso = NW * wbytes;
  return NW * wbytes <= kLdsLimit;
}

vbq_status launch_mm(const DevMatrix& m, uint32_t flags, const void* x, int64_t ldx, int M, void* y, int64_t ldy,
                     hipStream_t s) {
  int NW, S, lds;
  if (!mm_shape(m, &NW, &S, &lds)) return VBQ_ERR_UNSUPPORTED;
  MmArgs a;
  a.m = m;
  a.x = (const uint16_t*)x;
  a.y = y;
  a.ldx = ldx;
  a.ldy = ldy;
  a.M = M;
  a.S = S;
  a.yf16 = (flags & VBQ_Y_F16) ? 1 : 0;
  // row blocks of 16 per group: one, two or four (R = 16, 32, >= 64)
  if (m.R == 16) return launch_mm_rb<1>(a, NW, lds, s);
  if (m.R == 32) return launch_mm_rb<2>(a, NW, lds, s);
  return launch_mm_rb<4>(a, NW, lds, s);
}

// Name of the kernel a product with M activation rows launches on this matrix
// (the same choices as launch_mv / launch_mm); static storage.
// The one-launch plan of a bucketed GEMV (vbq_buckets_kernel<4>): every bucket
// a one-width matrix that the four-wave one-width kernel takes, two or more
// buckets, all with the same call options, every bucket's blob 256-byte
// aligned.  Buckets go smallest first, so their few tiles are dispatched
// with the first wave of workgroups.  False when the buckets do not qualify.
bool plan_buckets(const vbq_bucket* bk, int n, const void* blob, const int32_t* rows, BucketsArgs* ba, int* grid,
                  int* lds) {
  if (n < 2 || n > VBQ_MAX_BUCKETS) return false;
  int order[VBQ_MAX_BUCKETS];
  DevMatrix ms[VBQ_MAX_BUCKETS];
  for (int i = 0; i < n; ++i) {
    if (bk[i].desc.flags != bk[0].desc.flags || bk[i].row_begin < 0 || bk[i].n_rows != bk[i].desc.N) return false;
    if (make_dev_matrix(&bk[i].desc, (const uint8_t*)blob + bk[i].blob_offset, &ms[i]) != VBQ_OK) return false;
    order[i] = i;
  }
  std::sort(order, order + n, [&](int p, int q) { return ms[p].T != ms[q].T ? ms[p].T < ms[q].T : p < q; });
  *ba = BucketsArgs{};
  int tiles = 0, need = 0;
  for (int k = 0; k < n; ++k) {
    const int i = order[k];
    const DevMatrix& m = ms[i];
    int uni = -1, classes = 0;
    for (int c = 0; c < 4; ++c)
      if (m.n_entries[c]) {
        uni = c;
        ++classes;
      }
    MvShape sh;
    if (classes != 1 || !choose_shape(m, 1, &sh) || sh.NW != 4) return false;
    need = std::max(need, mv_lds_bytes(m.R, sh.SW, 1, 4, uni == 0 ? kLutBytes : 0, false));
    ba->m[k] = m;
    ba->rows[k] = rows + bk[i].row_begin;
    ba->tile0[k] = tiles;
    ba->cls[k] = uni;
    ba->S[k] = sh.S;
    ba->SW[k] = sh.SW;
    if ((int64_t)tiles + m.T > INT32_MAX) return false;
    tiles += (int)m.T;
  }
  if (need > kLdsLimit) return false;
  ba->n = n;
  ba->yf16 = (bk[0].desc.flags & VBQ_Y_F16) ? 1 : 0;
  *grid = tiles;
  *lds = need;
  return true;
}

const char* kernel_name(const DevMatrix& m, uint32_t flags, int M) {
  // (template arguments as the compiler prints them, spaces removed; the
  // uniform kernel's last argument is the width class log2 b)
  static const char* const kNames[] = {
      "vbq_mv_pair_kernel<8,1>", "vbq_mv_pair_kernel<16,1>", "vbq_mv_pair_kernel<8,2>",
      "vbq_mv_kernel<1,4>", "vbq_mv_kernel<1,8>", "vbq_mv_kernel<1,16>",
      "vbq_mv_kernel<2,4>", "vbq_mv_kernel<2,8>",
      "vbq_mv_kernel<1,4,0>", "vbq_mv_kernel<1,8,0>", "vbq_mv_kernel<1,16,0>",
      "vbq_mv_kernel<1,4,1>", "vbq_mv_kernel<1,8,1>", "vbq_mv_kernel<1,16,1>",
      "vbq_mv_kernel<1,4,2>", "vbq_mv_kernel<1,8,2>", "vbq_mv_kernel<1,16,2>",
      "vbq_mv_kernel<1,4,3>", "vbq_mv_kernel<1,8,3>", "vbq_mv_kernel<1,16,3>",
      "vbq_mm_kernel<4,1>", "vbq_mm_kernel<8,1>", "vbq_mm_kernel<16,1>",
      "vbq_mm_kernel<4,2>", "vbq_mm_kernel<8,2>", "vbq_mm_kernel<16,2>",
      "vbq_mm_kernel<4,4>", "vbq_mm_kernel<8,4>", "vbq_mm_kernel<16,4>",
      "none"};
  auto nw_index = [](int NW) { return NW == 4 ? 0 : NW == 8 ? 1 : 2; };
  if (M <= 0) return kNames[29];
  if (M <= 2) {
    if (!(flags & VBQ_ONE_WAVE_PER_UNIT)) {
      const int pw = pair_waves(m, M);
      if (pw) return kNames[M == 2 ? 2 : pw == 8 ? 0 : 1];
    }
    MvShape sh;
    if (!choose_shape(m, M, &sh)) return kNames[29];
    if (M == 2) return kNames[sh.NW == 4 ? 6 : 7];
    int uni = -1, classes = 0;
    for (int c = 0; c < 4; ++c)
      if (m.n_entries[c]) {
        uni = c;
        ++classes;
      }
    if (classes == 1) return kNames[8 + 3 * uni + nw_index(sh.NW)];
    return kNames[3 + nw_index(sh.NW)];
  }
  int NW, S, lds;
  if (!mm_shape(m, &NW, &S, &lds)) return kNames[29];
  const int rb = m.R == 16 ? 0 : m.R == 32 ? 1 : 2;
  return kNames[20 + 3 * rb + nw_index(NW)];
}

// ---------------------------------------------------------------------------
// One launch per decode step (paper section 6, "The speedup grows with model
// size": at small sizes the per-token overhead, not bandwidth, bounds decode).
//
// A step is a sequence of GEMVs in which GEMV i may read its x only once every
// earlier GEMV has written its y (in a model, x_i is computed from y_(i-1)).
// One persistent grid, one workgroup of 16 waves per CU, walks the sequence:
//   * GEMV i's row tiles are dealt to the workgroups in turn; a tile is worked
//     by wave pairs exactly as in vbq_mv_pair_kernel (the same per-entry
//     products, per-unit row sums and unit order, so y is bitwise the y of
//     the one-launch-per-GEMV path), two tiles at a time when they have at
//     most four units;
//   * the weights do not depend on x, so before waiting for GEMV i-1 a
//     workgroup issues the loads of its first tile of GEMV i (unit-table
//     rows, width map, the first code batch of every class) and builds the
//     entry index from the width map; only x, the decode, the row sums and
//     the stores of y follow the wait;
//   * a workgroup that has stored all its rows of GEMV i adds 1 to one of
//     eight arrival counters of GEMV i (eight words in eight 128-byte lines,
//     so the atomics do not all meet on one line); a workgroup waits for
//     GEMV i by polling the eight words until they sum to the number of
//     workgroups.
// Cross-workgroup visibility without cache flushes: y is written with
// device-coherent stores (agent scope), each wave waits until its stores have
// completed before its workgroup arrives, and x is read with device-coherent
// loads issued after the wait, so no release or acquire of the whole L2 is
// needed.  Waits are bounded: a workgroup that polls longer than the spin
// limit sets the status word, stops waiting and skips its remaining work
// (still arriving everywhere), so the grid always drains.
// ---------------------------------------------------------------------------
constexpr int kStepWaves = 16;
constexpr int kStepPairs = kStepWaves / 2;
constexpr int kStepSlots = 8;  // arrival words per GEMV
// words between two arrival words: each in its own 128-byte line, so the
// atomics and polls of different words do not queue on one line (measured on
// the 131M-class step: 614 us per step with the eight words in one line,
// 461 us with one line each)
constexpr int kStepSlotStride = 32;

struct StepOp {
  DevMatrix m;
  const uint16_t* x;
  void* y;
  const int32_t* rows;  // row map (as vbq_gemv_rows) or nullptr
  int64_t ylen;
  int32_t yf16;
  int32_t pad;
};

// x of one row for a window of `cols` group columns starting at column j,
// read with device-coherent loads (lanes past the window read the last chunk).
__device__ __forceinline__ void load_x1_coherent(const uint16_t* x, int K, int j, int cols, XRegs& xr,
                                                 uint32_t lane) {
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc((void*)x, 0, 2 * K, 0x00020000);
  const int n = cols * 8;
#pragma unroll
  for (int k = 0; k < kXRegs; ++k) {
    const int i = max(min((int)lane + 64 * k, n - 1), 0);
    // cache policy 16: the sc1 bit, the device-scope coherence of an agent-scope atomic load
    xr.v[k] = __builtin_amdgcn_raw_buffer_load_b128(r, 128 * j + 16 * i, 0, 16);
  }
}

__device__ __forceinline__ void store_y_coherent(void* y, size_t i, float v, int32_t f16) {
  if (f16)
    __hip_atomic_store((uint16_t*)y + i, __builtin_bit_cast(uint16_t, (_Float16)v), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  else
    __hip_atomic_store((float*)y + i, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Waits until GEMV `op` has n_wg arrivals (wave 0 polls the eight words,
// lanes 0..7 one each) or the spin limit is reached; every wave of the
// workgroup calls it and gets the result through LDS.  False on a timeout.
__device__ __forceinline__ bool step_wait(const uint32_t* sync, int op, uint32_t n_wg, uint32_t spin_limit,
                                          uint32_t flag_lds, int wave, uint32_t lane) {
  if (wave == 0) {
    const uint32_t* w = sync + ((size_t)op * kStepSlots + min(lane, (uint32_t)kStepSlots - 1)) * kStepSlotStride;
    uint32_t ok = 0;
    for (uint32_t it = 0; it < spin_limit; ++it) {
      const uint32_t v = lane < kStepSlots ? __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0u;
      if (wave_sum(v) >= n_wg) {
        ok = 1;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
    if (lane == 0) lds_store_f32(flag_lds, ok ? 1.0f : 0.0f);
  }
  __syncthreads();
  return lds_f32(flag_lds) != 0.0f;
}

// The arrival words of GEMV op: the unit to wait for when a later GEMV starts.
__global__ __launch_bounds__(kStepWaves * 64) void vbq_step_kernel(const StepOp* __restrict__ plan, int n_ops,
                                                                   uint32_t* __restrict__ sync,
                                                                   uint32_t* __restrict__ status,
                                                                   uint32_t spin_limit) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const uint32_t lds0 = (uint32_t)(size_t)(__attribute__((address_space(3))) uint8_t*)smem;
  const uint32_t flag_lds = lds0;  // 16 bytes: the wait's result
  const uint32_t base = lds0 + 16;
  const int wave = wave_id();
  // pair k = waves k and k + 8, which land on the same SIMD (see vbq_mv_pair_kernel)
  const int pair = wave % kStepPairs, role = wave / kStepPairs;
  const int wg = blockIdx.x, n_wg = gridDim.x;
  bool live = true;  // workgroup-uniform: false after a timed-out wait
  for (int op = 0; op < n_ops; ++op) {
    const StepOp* o = plan + op;
    DevMatrix mat = o->m;
    const int R = mat.R, U = mat.U, T = mat.T;
    const int tpr = U <= kStepPairs / 2 ? 2 : 1;  // tiles per round
    const int ups = kStepPairs / tpr;              // unit slots per tile
    const int slot = pair / ups, k = pair % ups;
    const WavePlan P = wave_plan(R, mat.C, 1);
    const uint32_t ysum0 = base;  // pair p's unit row sums at ysum0 + p*R*4
    const uint32_t ysum = ysum0 + (uint32_t)(pair * R * 4);
    const uint32_t region = base + (uint32_t)(kStepPairs * R * 4 + pair * P.bytes);
    Win wn;
    wn.xs = region + P.xs;
    wn.Xs = region + P.Xs;
    wn.part = region + P.part;
    wn.xstride_m = (uint32_t)(mat.C * kXStride);
    wn.part_m = (uint32_t)(mat.C * R * 4);
    wn.SW = mat.C;
    wn.logR = mat.logR;
    const uint32_t inv = region + P.inv;
    const int my_tiles = wg < T ? (T - wg + n_wg - 1) / n_wg : 0;
    const int rounds = (my_tiles + tpr - 1) / tpr;
    for (int rd = 0; rd < rounds; ++rd) {
      const uint32_t lane = lane_id_here();  // (values derived from it are not hoisted out of the loops)
      const int ti = rd * tpr + slot;
      const int t = wg + ti * n_wg;
      const bool active = ti < my_tiles && k < U;  // wave-uniform
      const bool must_wait = rd == 0 && op > 0;    // workgroup-uniform
      const UnitInfo u = load_unit(mat, active ? t : 0, active ? k : 0);
      const int unit = (active ? t : 0) * mat.U + (active ? k : 0);
      uint32_t start[4], seg[4];
      int n[4];
      WinCounts wc;
      // The two roles run separate code paths with the same sequence of
      // workgroup barriers, so each keeps only its own batches in registers.
      if (role == 0) {
        // ---- before the wait: what depends on the weights only
        for (int i = (int)lane; i < R; i += 64) lds_store_f32(ysum + 4u * i, 0.0f);
        Batch<0, 1> A0;
        if (active && live) {
          const WmapRegs wr = load_wmap(mat, u, u.W, lane);
          const u32x16 rows2 = unit_rows(mat, unit);
          const u32x4 erow = rows2.s0123, own = rows2.s89ab - rows2.s0123;
          wc.own[0] = own.x;
          wc.own[1] = own.y;
          wc.own[2] = own.z;
          wc.own[3] = own.w;
          const uint32_t es[4] = {erow.x, erow.y, erow.z, erow.w};
          uint32_t acc = 0;
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            // (wave-uniform values, kept in scalar registers: the decode's vector
            // registers are the step kernel's tightest resource)
            wc.before[c] = 0u;
            start[c] = (uint32_t)uniform((int)es[c]);
            n[c] = uniform(clamp_run(mat, c, start[c], (uint32_t)uniform((int)wc.own[c])));
            seg[c] = (uint32_t)uniform((int)(inv + 2u * acc));
            acc += (uint32_t)uniform((int)wc.own[c]);
          }
          load_batch<0, 1>(A0, mat, start[0], n[0], 0, lane);
          build_index(wr, u, 0, u.W, R, wc, inv, lane);
        }
        if (must_wait && live && !step_wait(sync, op - 1, (uint32_t)n_wg, spin_limit, flag_lds, wave, lane)) {
          live = false;
          if (wave == 0 && lane == 0) __hip_atomic_store(status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        __syncthreads();  // the index and x of every unit are in LDS
        if (active && live) run_class<0, 1>(mat, A0, start[0], n[0], seg[0], wn, lane);
        __syncthreads();  // every partial product is in LDS
        if (active && live) reduce_window<1>(wn, R, u.cols, u.rows, ysum, lane);
        __syncthreads();
      } else {
        Batch<1, 1> A1;
        Batch<2, 1> A2;
        Batch<3, 1> A3;
        if (active && live) {
          const u32x16 rows2 = unit_rows(mat, unit);
          const u32x4 erow = rows2.s0123, own = rows2.s89ab - rows2.s0123;
          const uint32_t es[4] = {erow.x, erow.y, erow.z, erow.w};
          const uint32_t ow[4] = {own.x, own.y, own.z, own.w};
          uint32_t acc = 0;
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            start[c] = (uint32_t)uniform((int)es[c]);
            n[c] = uniform(clamp_run(mat, c, start[c], (uint32_t)uniform((int)ow[c])));
            seg[c] = (uint32_t)uniform((int)(inv + 2u * acc));
            acc += (uint32_t)uniform((int)ow[c]);
          }
          load_batch<1, 1>(A1, mat, start[1], n[1], 0, lane);
          load_batch<2, 1>(A2, mat, start[2], n[2], 0, lane);
        }
        if (must_wait && live && !step_wait(sync, op - 1, (uint32_t)n_wg, spin_limit, flag_lds, wave, lane))
          live = false;
        if (active && live) {
          XRegs xr;
          load_x1_coherent(o->x, mat.K, u.j0, u.cols, xr, lane);
          store_x1(u.cols, xr, wn, lane);
        }
        __syncthreads();  // the index and x of every unit are in LDS
        if (active && live) {
          run_class<1, 1>(mat, A1, start[1], n[1], seg[1], wn, lane);
          run_class<2, 1>(mat, A2, start[2], n[2], seg[2], wn, lane);
          // the 8-bit batch only now: held across the other classes' decode it
          // made the kernel spill (one 1 KB scratch round trip per decoded slot)
          load_batch<3, 1>(A3, mat, start[3], n[3], 0, lane);
          run_class<3, 1>(mat, A3, start[3], n[3], seg[3], wn, lane);
        }
        __syncthreads();  // every partial product is in LDS
        __syncthreads();  // (role 0 adds the row sums)
      }
      // per tile slot: the unit row sums added in unit order, stored coherently
      for (int i = threadIdx.x; i < tpr * R; i += kStepWaves * 64) {
        const int sl = i / R, r = i - sl * R;
        const int tt = wg + (rd * tpr + sl) * n_wg;
        if (live && rd * tpr + sl < my_tiles && r < min(R, mat.N - tt * R)) {
          float tot = 0.0f;
          for (int kk = 0; kk < U; ++kk) tot += lds_f32(ysum0 + 4u * (uint32_t)((sl * ups + kk) * R + r));
          const size_t row = (size_t)tt * R + r;
          if (o->rows == nullptr) {
            store_y_coherent(o->y, row, tot, o->yf16);
          } else {
            const int64_t d = o->rows[row];
            if (d >= 0 && d < o->ylen) store_y_coherent(o->y, (size_t)d, tot, o->yf16);
          }
        }
      }
      __syncthreads();  // LDS is reused by the next round
    }
    // arrival: every wave's stores of y have completed, then one atomic
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0)
      __hip_atomic_fetch_add(sync + ((size_t)op * kStepSlots + (wg & (kStepSlots - 1))) * kStepSlotStride, 1u,
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Clears the arrival words and the status word before a step.
__global__ __launch_bounds__(256) void vbq_step_clear_kernel(uint32_t* sync, uint32_t words, uint32_t* status) {
  for (uint32_t i = threadIdx.x + blockIdx.x * 256u; i < words; i += 256u * gridDim.x) sync[i] = 0u;
  if (threadIdx.x == 0 && blockIdx.x == 0) *status = 0u;
}

// Bytes of LDS one step-kernel workgroup needs for a matrix (16-byte flag,
// then eight pairs' row sums and regions).
inline int step_lds_bytes(const DevMatrix& m) {
  return 16 + kStepPairs * (m.R * 4 + wave_plan(m.R, m.C, 1).bytes);
}

uint32_t step_arrival_words(int n) { return (uint32_t)n * kStepSlots * kStepSlotStride; }
uint32_t step_sync_words(int n) { return step_arrival_words(n) + 1u; }  // + the status word

vbq_status launch_step(const void* plan_dev, int32_t n, uint32_t* sync, uint32_t* status, uint32_t spin_limit,
                       void* stream);

// Scratch of vbq_step_run_noalloc: the arrival words and the status word of a
// step of up to kNoAllocMaxGemvs GEMVs (512 KiB; every GPU the library runs on
// holds its own copy until the process ends).  Host code never uses this name
// as an address: it is a host-side stand-in, and the device address comes from
// hipGetSymbolAddress, once per device.
constexpr int kNoAllocMaxGemvs = 512;
constexpr int kNoAllocWords = kNoAllocMaxGemvs * kStepSlots * kStepSlotStride + 64;
static __device__ __align__(256) uint32_t scratch[kNoAllocWords];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint32_t* g_scratch_dev[kMaxDevices] = {};

// The current device's copy of `scratch`, looked up on the first call per device.
vbq_status scratch_address(uint32_t** out) {
  int dev = 0;
  vbq_status st = hip_status(hipGetDevice(&dev));
  if (st != VBQ_OK) return st;
  if (dev < 0 || dev >= kMaxDevices) return VBQ_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    st = hip_status(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (st != VBQ_OK) return st;
    if (!p) return VBQ_ERR_HIP;
    g_scratch_dev[dev] = (uint32_t*)p;
  }
  *out = g_scratch_dev[dev];
  return VBQ_OK;
}

}  // namespace

// Shared with the other device sources of the library: records a failed HIP
// call for vbq_last_hip_error and maps it to a status.
vbq_status vbq_detail_hip_status(hipError_t e) { return hip_status(e); }

extern "C" {

const char* vbq_last_hip_error(void) { return hipGetErrorName(g_last_hip_error); }

// Required alignment of y: 4 bytes for float, 2 for fp16.
inline uintptr_t y_align(const vbq_desc* d) { return (d->flags & VBQ_Y_F16) ? 2 : 4; }

vbq_status vbq_gemv(const vbq_desc* desc, const void* blob_dev, const void* x_dev, void* y_dev, void* stream) {
  if (!x_dev || !y_dev) return VBQ_ERR_NULL;
  DevMatrix m;
  vbq_status st = make_dev_matrix(desc, blob_dev, &m);
  if (st != VBQ_OK) return st;
  if ((uintptr_t)x_dev % 16 || (uintptr_t)y_dev % y_align(desc)) return VBQ_ERR_BUFFER;
  return launch_mv<1>(m, desc->flags, x_dev, desc->K, 1, y_dev, desc->N, (hipStream_t)stream);
}

vbq_status vbq_gemv_rows(const vbq_desc* desc, const void* blob_dev, const void* x_dev, void* y_dev, int64_t y_len,
                         const int32_t* row_index_dev, void* stream) {
  if (!x_dev || !y_dev || !row_index_dev) return VBQ_ERR_NULL;
  if (y_len < 0) return VBQ_ERR_SHAPE;
  DevMatrix m;
  vbq_status st = make_dev_matrix(desc, blob_dev, &m);
  if (st != VBQ_OK) return st;
  if ((uintptr_t)x_dev % 16 || (uintptr_t)y_dev % y_align(desc) || (uintptr_t)row_index_dev % 4)
    return VBQ_ERR_BUFFER;
  return launch_mv<1>(m, desc->flags, x_dev, desc->K, 1, y_dev, desc->N, (hipStream_t)stream, row_index_dev, y_len);
}

vbq_status vbq_gemv_buckets(const vbq_bucket* buckets, int32_t n_buckets, const void* blob_dev,
                            const int32_t* row_index_dev, const void* x_dev, void* y_dev, int64_t y_len,
                            void* stream) {
  if (n_buckets < 0 || n_buckets > VBQ_MAX_BUCKETS) return VBQ_ERR_SHAPE;
  if (n_buckets == 0) return VBQ_OK;
  if (!buckets || !blob_dev || !row_index_dev) return VBQ_ERR_NULL;
  for (int32_t i = 0; i < n_buckets; ++i) {
    const vbq_bucket& b = buckets[i];
    if (b.row_begin < 0 || b.n_rows != b.desc.N) return VBQ_ERR_DESC;
  }
  if (x_dev && y_dev && y_len >= 0 && (uintptr_t)x_dev % 16 == 0 && (uintptr_t)row_index_dev % 4 == 0) {
    BucketsArgs ba;
    int grid = 0, lds = 0;
    if (plan_buckets(buckets, n_buckets, blob_dev, row_index_dev, &ba, &grid, &lds) &&
        (uintptr_t)y_dev % y_align(&buckets[0].desc) == 0) {
      ba.x = (const uint16_t*)x_dev;
      ba.y = y_dev;
      ba.ylen = y_len;
      const void* kernel = (const void*)vbq_buckets_kernel<4>;
      if (lds > 64 * 1024) {
        static std::atomic<uint64_t> done{0};
        vbq_status st = allow_big_lds(kernel, done);
        if (st != VBQ_OK) return st;
      }
      void* kargs[] = {&ba};
      return hip_status(hipLaunchKernel(kernel, dim3((unsigned)grid), dim3(4 * 64), kargs, (size_t)lds,
                                        (hipStream_t)stream));
    }
  }
  // otherwise (and for every argument error) one vbq_gemv_rows per bucket
  for (int32_t i = 0; i < n_buckets; ++i) {
    const vbq_bucket& b = buckets[i];
    const vbq_status st = vbq_gemv_rows(&b.desc, (const uint8_t*)blob_dev + b.blob_offset, x_dev, y_dev, y_len,
                                        row_index_dev + b.row_begin, stream);
    if (st != VBQ_OK) return st;
  }
  return VBQ_OK;
}

const char* vbq_gemv_buckets_kernel_name(const vbq_bucket* buckets, int32_t n_buckets) {
  if (n_buckets < 1 || n_buckets > VBQ_MAX_BUCKETS || !buckets) return "none";
  BucketsArgs ba;
  int grid = 0, lds = 0;
  // (any aligned non-null addresses: only the descriptors are looked at)
  if (plan_buckets(buckets, n_buckets, (const void*)(uintptr_t)256, (const int32_t*)(uintptr_t)256, &ba, &grid, &lds))
    return "vbq_buckets_kernel<4>";
  return "per bucket";
}

vbq_status vbq_gemm_small(const vbq_desc* desc, const void* blob_dev, int64_t M, const void* X_dev, int64_t ldx,
                          void* Y_dev, int64_t ldy, void* stream) {
  if (M < 0 || M > VBQ_MAX_M) return VBQ_ERR_SHAPE;
  DevMatrix m;
  vbq_status st = make_dev_matrix(desc, blob_dev, &m);
  if (st != VBQ_OK) return st;
  if (M == 0) return VBQ_OK;
  if (!X_dev || !Y_dev) return VBQ_ERR_NULL;
  if (ldx < desc->K || ldx % 8 || ldy < desc->N) return VBQ_ERR_SHAPE;
  if ((uintptr_t)X_dev % 16 || (uintptr_t)Y_dev % y_align(desc)) return VBQ_ERR_BUFFER;
  hipStream_t s = (hipStream_t)stream;
  const int Mi = (int)M;
  const uint32_t f = desc->flags;
  if (Mi == 1) return launch_mv<1>(m, f, X_dev, ldx, 1, Y_dev, ldy, s);
  if (Mi == 2) return launch_mv<2>(m, f, X_dev, ldx, 2, Y_dev, ldy, s);
  return launch_mm(m, f, X_dev, ldx, Mi, Y_dev, ldy, s);
}

const char* vbq_kernel_name(const vbq_desc* desc, int64_t M) {
  DevMatrix m;
  // (any aligned non-null address: only the descriptor is looked at)
  if (!desc || make_dev_matrix(desc, (const void*)(uintptr_t)256, &m) != VBQ_OK || M < 0 || M > VBQ_MAX_M)
    return "none";
  return kernel_name(m, desc->flags, (int)M);
}

vbq_status vbq_dequant(const vbq_desc* desc, const void* blob_dev, float* W_dev, void* stream) {
  if (!W_dev) return VBQ_ERR_NULL;
  DevMatrix m;
  vbq_status st = make_dev_matrix(desc, blob_dev, &m);
  if (st != VBQ_OK) return st;
  if ((uintptr_t)W_dev % 4) return VBQ_ERR_BUFFER;
  // one uint16 per position of the widest wave slice, rounded up to whole words
  int region = align16(((max_slice_cols(m.R, m.C, kDequantWaves) * m.R + 63) / 64) * 64 * 2);
  void* args[] = {&m, &W_dev, &region};
  const int lds = kDequantWaves * region;
  return hip_status(hipLaunchKernel((const void*)vbq_dequant_kernel, dim3((unsigned)m.T), dim3(kDequantWaves * 64), args,
                                    (size_t)lds, (hipStream_t)stream));
}

vbq_status vbq_step_plan_bytes(int32_t n, size_t* bytes) {
  if (!bytes) return VBQ_ERR_NULL;
  if (n < 1 || n > VBQ_STEP_MAX_GEMVS) return VBQ_ERR_SHAPE;
  *bytes = (size_t)n * sizeof(StepOp);
  return VBQ_OK;
}

vbq_status vbq_step_workspace_bytes(int32_t n, size_t* bytes) {
  if (!bytes) return VBQ_ERR_NULL;
  if (n < 1 || n > VBQ_STEP_MAX_GEMVS) return VBQ_ERR_SHAPE;
  *bytes = (size_t)step_sync_words(n) * 4;
  return VBQ_OK;
}

vbq_status vbq_step_plan(const vbq_step_gemv* gemvs, int32_t n, void* plan_host, size_t plan_bytes) {
  if (!gemvs || !plan_host) return VBQ_ERR_NULL;
  if (n < 1 || n > VBQ_STEP_MAX_GEMVS) return VBQ_ERR_SHAPE;
  if (plan_bytes < (size_t)n * sizeof(StepOp) || (uintptr_t)plan_host % 8) return VBQ_ERR_BUFFER;
  StepOp* ops = (StepOp*)plan_host;
  for (int32_t i = 0; i < n; ++i) {
    const vbq_step_gemv& g = gemvs[i];
    if (!g.desc || !g.x || !g.y) return VBQ_ERR_NULL;
    StepOp op{};
    vbq_status st = make_dev_matrix(g.desc, g.blob, &op.m);
    if (st != VBQ_OK) return st;
    if (g.desc->flags & VBQ_ONE_WAVE_PER_UNIT) return VBQ_ERR_UNSUPPORTED;
    // the tile body is the wave-pair one: at most eight units of at most 32 columns
    if (op.m.U > kStepPairs || op.m.C > kXRegs * 8 || step_lds_bytes(op.m) > kLdsLimit) return VBQ_ERR_UNSUPPORTED;
    if ((uintptr_t)g.x % 16 || (uintptr_t)g.y % y_align(g.desc)) return VBQ_ERR_BUFFER;
    if (g.rows && ((uintptr_t)g.rows % 4 || g.y_len < 0)) return g.y_len < 0 ? VBQ_ERR_SHAPE : VBQ_ERR_BUFFER;
    op.x = (const uint16_t*)g.x;
    op.y = g.y;
    op.rows = g.rows;
    op.ylen = g.rows ? g.y_len : 0;
    op.yf16 = (g.desc->flags & VBQ_Y_F16) ? 1 : 0;
    ops[i] = op;
  }
  return VBQ_OK;
}

vbq_status vbq_step_run(const void* plan_dev, int32_t n, void* workspace_dev, size_t workspace_bytes,
                        uint32_t spin_limit, void* stream) {
  if (!plan_dev || !workspace_dev) return VBQ_ERR_NULL;
  if (n < 1 || n > VBQ_STEP_MAX_GEMVS) return VBQ_ERR_SHAPE;
  const uint32_t words = step_sync_words(n);
  if (workspace_bytes < (size_t)words * 4 || (uintptr_t)workspace_dev % 4 || (uintptr_t)plan_dev % 8)
    return VBQ_ERR_BUFFER;
  uint32_t* sync = (uint32_t*)workspace_dev;
  return launch_step(plan_dev, n, sync, sync + step_arrival_words(n), spin_limit, stream);
}

vbq_status vbq_step_run_noalloc(const void* plan_dev, int32_t n, uint32_t spin_limit, uint32_t* status_dev,
                                void* stream) {
  if (!plan_dev) return VBQ_ERR_NULL;
  if (n < 1 || n > kNoAllocMaxGemvs) return VBQ_ERR_SHAPE;
  if ((uintptr_t)plan_dev % 8 || (uintptr_t)status_dev % 4) return VBQ_ERR_BUFFER;
  uint32_t* sync = nullptr;
  vbq_status st = scratch_address(&sync);
  if (st != VBQ_OK) return st;
  // the status word: the caller's, or the last word of the scratch
  return launch_step(plan_dev, n, sync, status_dev ? status_dev : sync + (kNoAllocWords - 1), spin_limit, stream);
}

}  // extern "C"

namespace {

// The clearing kernel and the cooperative launch of the step kernel over the
// arrival words `sync` (step_arrival_words(n) words) and the status word.
vbq_status launch_step(const void* plan_dev, int32_t n, uint32_t* sync, uint32_t* status, uint32_t spin_limit,
                       void* stream) {
  if (spin_limit == 0) spin_limit = 1u << 22;
  const uint32_t words = step_arrival_words(n);
  const void* kernel = (const void*)vbq_step_kernel;
  static std::atomic<uint64_t> done{0};
  vbq_status st = allow_big_lds(kernel, done);
  if (st != VBQ_OK) return st;
  // one workgroup of 16 waves per CU, all resident at once (checked here, and
  // the cooperative launch refuses a grid that does not fit)
  int dev = 0, cus = 0, per_cu = 0;
  if ((st = hip_status(hipGetDevice(&dev))) != VBQ_OK) return st;
  if ((st = hip_status(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev))) != VBQ_OK) return st;
  const size_t lds = kLdsLimit;
  if ((st = hip_status(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kStepWaves * 64, lds))) !=
      VBQ_OK)
    return st;
  if (per_cu < 1 || cus < 1) return VBQ_ERR_UNSUPPORTED;
  const unsigned grid = (unsigned)cus;
  hipStream_t s = (hipStream_t)stream;
  {
    void* args[] = {&sync, (void*)&words, &status};
    st = hip_status(hipLaunchKernel((const void*)vbq_step_clear_kernel, dim3(1), dim3(256), args, 0, s));
    if (st != VBQ_OK) return st;
  }
  const StepOp* plan = (const StepOp*)plan_dev;
  int nops = n;
  void* args[] = {&plan, &nops, &sync, &status, &spin_limit};
  return hip_status(hipLaunchCooperativeKernel(kernel, dim3(grid), dim3(kStepWaves * 64), args, lds, s));
}

}  // namespace
