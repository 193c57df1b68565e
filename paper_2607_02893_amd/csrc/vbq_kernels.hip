// Fused dequantize-and-multiply over packed variable-bit-width weights, for
// gfx950 (MI355X).  Paper section 6 ("Fused kernels over packed weights"):
// every group's packed codes are expanded in registers with the group scale
// and accumulated, so the full-precision matrix never exists in memory.
//
// Work decomposition (layout version 1, include/vbq.h):
//   * one workgroup (256 lanes, 4 wave64) owns a row tile and walks its
//     column-chunk units in order;
//   * per unit it rebuilds, in LDS, the position of every entry of each width
//     class from the 2-bit width map (ballot-free: word popcounts, a wave scan
//     and mbcnt), so lanes can be handed 64 consecutive entries of ONE width;
//   * each lane decodes one 64-weight group with width-specific, branch-free
//     bit tricks: a masked field of codes, read as a pair of fp16 values, is a
//     power-of-two multiple of the codes, so v_dot2_f32_f16 multiplies two
//     weights by their activations in one instruction and the power of two is
//     folded in once per group;
//   * the offset of the offset-binary codes is removed with the group's
//     activation sum X_j = sum x: sum q x = sum u x - 2^(b-1) X_j (b >= 2),
//     sum q x = 2 sum u x - X_j (b = 1);
//   * per-group partial results go to LDS at their (row, column) position and
//     each row is summed in a fixed order, so results are bitwise repeatable.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "vbq_layout.hpp"

namespace {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kMaxWords = vbq::kMaxUnitPositions / 64;  // width-map words per plane of a unit

struct DevMatrix {
  const uint32_t* units;
  const uint64_t* wmap;
  const uint8_t* codes[4];
  const uint16_t* scales[4];
  uint32_t n_entries[4];
  int32_t N, K, G, R, C, T, U, logR;
};

struct MvArgs {
  DevMatrix m;
  const uint16_t* x;  // fp16 bits, row m at x + m*ldx
  float* y;           // row m at y + m*ldy
  int64_t ldx, ldy;
  int32_t M;          // rows of x actually present (<= MT)
  int32_t SC;         // group columns per sub-chunk (LDS staging window)
};

__device__ __forceinline__ half2_t as_h2(uint32_t v) { return __builtin_bit_cast(half2_t, v); }

__device__ __forceinline__ float dot2(uint32_t codes, uint32_t xpair, float acc) {
  return __builtin_amdgcn_fdot2(as_h2(codes), as_h2(xpair), acc, false);
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

// ---------------------------------------------------------------------------
// Index build: positions of each class's entries inside one unit.
// ---------------------------------------------------------------------------
struct UnitInfo {
  int j0, cols, rows, npos, W;      // first group column, columns, real rows, positions, words/plane
  uint32_t start[4];               // first global entry of each class
  int n[4];                        // entries of each class in the unit
  int base[4];                     // class segment start inside inv[]
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
  const int unit = t * mat.U + k;
  u.j0 = k * mat.C;
  u.cols = min(mat.C, mat.G - u.j0);
  u.rows = min(mat.R, mat.N - t * mat.R);
  u.npos = u.cols * mat.R;
  u.W = (u.npos + 63) >> 6;
  const uint32_t* row = mat.units + (size_t)unit * vbq::kUnitRowWords;
  const uint32_t* nxt = row + vbq::kUnitRowWords;
  int base = 0;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    u.start[c] = row[c];
    uint32_t end = nxt[c];
    // never step outside the class section, whatever the blob says
    if (end > mat.n_entries[c]) end = mat.n_entries[c];
    int n = end > u.start[c] ? (int)(end - u.start[c]) : 0;
    if (n > u.npos - base) n = u.npos - base;  // segments of inv[] stay inside R*C
    u.n[c] = n;
    u.base[c] = base;
    base += n;
  }
  u.wmap_word = row[4];
  return u;
}

// Builds inv[base[c] + e] = position of the e-th class-c entry, and
// pre[c][w] = number of class-c entries in words < w (w = 0..W).
__device__ void build_index(const DevMatrix& mat, const UnitInfo& u, uint16_t* inv, uint16_t (*pre)[kMaxWords + 1]) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint64_t* plane0 = mat.wmap + u.wmap_word;
  const uint64_t* plane1 = plane0 + u.W;
  // phase A: class counts per word (one thread per word)
  for (int w = tid; w < u.W; w += kThreads) {
    uint64_t m[4];
    class_masks(plane0[w], plane1[w], valid_mask(w, u.npos, mat.R, u.rows), m);
#pragma unroll
    for (int c = 0; c < 4; ++c) pre[c][w + 1] = (uint16_t)__popcll(m[c]);
  }
  __syncthreads();
  // phase B: inclusive scan over words, wave 0 (each lane owns two words)
  if (wave == 0) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int w0 = 2 * lane, w1 = 2 * lane + 1;
      const int a = w0 < u.W ? pre[c][w0 + 1] : 0;
      const int b = w1 < u.W ? pre[c][w1 + 1] : 0;
      int incl = a + b;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const int o = __shfl_up(incl, d, 64);
        if (lane >= d) incl += o;
      }
      const int excl = incl - a - b;
      if (w0 < u.W) pre[c][w0 + 1] = (uint16_t)(excl + a);
      if (w1 < u.W) pre[c][w1 + 1] = (uint16_t)(excl + a + b);
      if (lane == 0) pre[c][0] = 0;
    }
  }
  __syncthreads();
  // phase C: every wave takes whole words; lanes are positions
  for (int w = wave; w < u.W; w += kWaves) {
    uint64_t m[4];
    const uint64_t p0 = plane0[w], p1 = plane1[w];
    class_masks(p0, p1, valid_mask(w, u.npos, mat.R, u.rows), m);
    const int c = (int)((p0 >> lane) & 1) | ((int)((p1 >> lane) & 1) << 1);
    const uint64_t mine = c == 0 ? m[0] : c == 1 ? m[1] : c == 2 ? m[2] : m[3];
    if ((mine >> lane) & 1) {
      const int rank = pre[c][w] + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mine >> 32),
                                                                 __builtin_amdgcn_mbcnt_lo((uint32_t)mine, 0u));
      if (rank < u.n[c]) inv[u.base[c] + rank] = (uint16_t)(w * 64 + lane);
    }
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// Per-class fused decode + multiply for a window of group columns.
// ---------------------------------------------------------------------------
template <int CLS, int MT>
__device__ __forceinline__ void mv_class(const MvArgs& a, const UnitInfo& u, const uint16_t* inv,
                                         const uint16_t (*pre)[kMaxWords + 1], int wlo, int whi, int js0,
                                         int scols, const u32x4* xs, const float* Xs, float* part) {
  using D = Dec<CLS>;
  constexpr int NW = 2 * D::B;  // uint32 words per entry
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int e_lo = pre[CLS][wlo], e_hi = min((int)pre[CLS][whi], u.n[CLS]);
  const uint32_t* codes = (const uint32_t*)a.m.codes[CLS];
  const uint16_t* scales = a.m.scales[CLS];
  const int R = a.m.R, logR = a.m.logR;
  const int plane = scols * R;  // partials per x row in this window
  for (int e0 = e_lo + wave * 64; e0 < e_hi; e0 += kWaves * 64) {
    const int e = e0 + lane;
    if (e >= e_hi) continue;
    const int p = inv[u.base[CLS] + e];
    const int js = (p >> logR) - js0;     // column inside the window
    const int r = p & (R - 1);
    const size_t g = (size_t)u.start[CLS] + e;
    uint32_t w[NW];
    if constexpr (NW == 2) {
      const u32x2 v = __builtin_nontemporal_load((const u32x2*)(codes + g * NW));
      w[0] = v.x;
      w[1] = v.y;
    } else {
#pragma unroll
      for (int i = 0; i < NW / 4; ++i) {
        const u32x4 v = __builtin_nontemporal_load((const u32x4*)(codes + g * NW) + i);
        w[4 * i] = v.x;
        w[4 * i + 1] = v.y;
        w[4 * i + 2] = v.z;
        w[4 * i + 3] = v.w;
      }
    }
    const float s = (float)__builtin_bit_cast(_Float16, scales[g]);
    float acc[MT][D::kSlots];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int k = 0; k < D::kSlots; ++k) acc[m][k] = 0.0f;
#pragma unroll
    for (int q = 0; q < 8; ++q) {  // x chunk q holds pairs 4q..4q+3
      u32x4 xv[MT];
#pragma unroll
      for (int m = 0; m < MT; ++m) xv[m] = xs[(m * 8 + q) * scols + js];
#pragma unroll
      for (int c4 = 0; c4 < 4; ++c4) {
        const int i = 4 * q + c4;                  // pair index
        const int wi = i / D::kFields, f = i % D::kFields;
        constexpr uint32_t one = (1u << D::B) - 1;
        const Field fd = D::field(f);
        const uint32_t mask = (one << fd.t) * 0x00010001u;
        const uint32_t v = shl(w[wi], fd.shift) & mask;
        const int sl = D::slot(fd.t);
#pragma unroll
        for (int m = 0; m < MT; ++m) acc[m][sl] = dot2(v, xv[m][c4], acc[m][sl]);
      }
    }
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      float su = acc[m][0] * D::inv_value(0);
#pragma unroll
      for (int k = 1; k < D::kSlots; ++k) su = __builtin_fmaf(acc[m][k], D::inv_value(k), su);
      const float X = Xs[m * scols + js];
      const float sq = CLS == 0 ? __builtin_fmaf(su, 2.0f, -X) : __builtin_fmaf(-(float)(1 << (D::B - 1)), X, su);
      part[m * plane + js * R + r] = s * sq;
    }
  }
}

// Stage x for group columns [j0, j0+cols) of every present row into LDS as
// 16-byte chunks, chunk-major: xs[(m*8 + q)*cols + j] = x[m][(j0+j)*64 + 8q .. +8].
// Then Xs[m*cols + j] = sum of the 64 activations of column j, in fixed order.
template <int MT>
__device__ __forceinline__ void stage_x(const MvArgs& a, int j0, int cols, u32x4* xs, float* Xs) {
  const int tid = threadIdx.x;
  const int n = MT * cols * 8;
  for (int i = tid; i < n; i += kThreads) {
    const int m = i / (cols * 8), rem = i - m * cols * 8, j = rem >> 3, q = rem & 7;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (m < a.M) v = *(const u32x4*)(a.x + m * a.ldx + (size_t)(j0 + j) * 64 + q * 8);
    xs[(m * 8 + q) * cols + j] = v;
  }
  __syncthreads();
  const uint32_t ones = 0x3C003C00u;  // (1.0, 1.0)
  for (int i = tid; i < MT * cols; i += kThreads) {
    const int m = i / cols, j = i - m * cols;
    float acc = 0.0f;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const u32x4 v = xs[(m * 8 + q) * cols + j];
      acc = dot2(v.x, ones, acc);
      acc = dot2(v.y, ones, acc);
      acc = dot2(v.z, ones, acc);
      acc = dot2(v.w, ones, acc);
    }
    Xs[i] = acc;
  }
  __syncthreads();
}

struct LdsPlan {
  int inv, pre, xs, Xs, part, yacc, red, total;
};

__host__ __device__ inline int align16(int v) { return (v + 15) & ~15; }

__host__ __device__ inline LdsPlan lds_plan(int R, int C, int MT, int SC) {
  LdsPlan p;
  int o = 0;
  p.inv = o;  o += align16(R * C * 2);
  p.pre = o;  o += align16(4 * (kMaxWords + 1) * 2);
  p.xs = o;   o += MT * 8 * SC * 16;
  p.Xs = o;   o += align16(MT * SC * 4);
  p.part = o; o += align16(MT * SC * R * 4);
  p.yacc = o; o += align16(MT * R * 4);
  p.red = o;  o += kThreads * 4;
  p.total = o;
  return p;
}

template <int MT>
__global__ __launch_bounds__(kThreads) void vbq_mv_kernel(MvArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const DevMatrix& mat = a.m;
  const LdsPlan L = lds_plan(mat.R, mat.C, MT, a.SC);
  uint16_t* inv = (uint16_t*)(smem + L.inv);
  auto pre = (uint16_t(*)[kMaxWords + 1])(smem + L.pre);
  u32x4* xs = (u32x4*)(smem + L.xs);
  float* Xs = (float*)(smem + L.Xs);
  float* part = (float*)(smem + L.part);
  float* yacc = (float*)(smem + L.yacc);
  float* red = (float*)(smem + L.red);
  const int tid = threadIdx.x;
  const int R = mat.R;
  const int NS = MT * R;  // output slots (x row, tile row)

  for (int t = blockIdx.x; t < mat.T; t += gridDim.x) {
    for (int i = tid; i < NS; i += kThreads) yacc[i] = 0.0f;
    for (int k = 0; k < mat.U; ++k) {
      const UnitInfo u = load_unit(mat, t, k);
      build_index(mat, u, inv, pre);
      for (int js0 = 0; js0 < u.cols; js0 += a.SC) {
        const int scols = min(a.SC, u.cols - js0);
        // words covering positions [js0*R, (js0+scols)*R): SC*R is a multiple of 64
        const int wlo = (js0 * R) >> 6, whi = min(u.W, ((js0 + scols) * R + 63) >> 6);
        stage_x<MT>(a, u.j0 + js0, scols, xs, Xs);
        mv_class<0, MT>(a, u, inv, pre, wlo, whi, js0, scols, xs, Xs, part);
        mv_class<1, MT>(a, u, inv, pre, wlo, whi, js0, scols, xs, Xs, part);
        mv_class<2, MT>(a, u, inv, pre, wlo, whi, js0, scols, xs, Xs, part);
        mv_class<3, MT>(a, u, inv, pre, wlo, whi, js0, scols, xs, Xs, part);
        __syncthreads();
        // fixed-order row sums of this window: S threads per slot, then S partials in order
        const int plane = scols * R;
        if (NS <= kThreads) {
          const int S = kThreads / NS;  // NS and kThreads are powers of two
          const int slot = tid % NS, sub = tid / NS;
          const int m = slot / R, r = slot % R;
          float acc = 0.0f;
          if (r < u.rows)
            for (int j = sub; j < scols; j += S) acc += part[m * plane + j * R + r];
          red[tid] = acc;
          __syncthreads();
          if (tid < NS && r < u.rows) {
            float tot = 0.0f;
            for (int s2 = 0; s2 < S; ++s2) tot += red[s2 * NS + slot];
            yacc[slot] += tot;
          }
        } else {
          for (int slot = tid; slot < NS; slot += kThreads) {
            const int m = slot / R, r = slot % R;
            if (r >= u.rows) continue;
            float acc = 0.0f;
            for (int j = 0; j < scols; ++j) acc += part[m * plane + j * R + r];
            yacc[slot] += acc;
          }
        }
        __syncthreads();
      }
    }
    const int rows = min(R, mat.N - t * R);
    for (int slot = tid; slot < NS; slot += kThreads) {
      const int m = slot / R, r = slot % R;
      if (m < a.M && r < rows) a.y[m * a.ldy + (size_t)t * R + r] = yacc[slot];
    }
    __syncthreads();
  }
}

// w_hat = s*q written densely, one lane per entry (checking aid, not a hot path).
__global__ __launch_bounds__(kThreads) void vbq_dequant_kernel(DevMatrix mat, float* W) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  uint16_t* inv = (uint16_t*)smem;
  auto pre = (uint16_t(*)[kMaxWords + 1])(smem + align16(mat.R * mat.C * 2));
  for (int t = blockIdx.x; t < mat.T; t += gridDim.x) {
    for (int k = 0; k < mat.U; ++k) {
      const UnitInfo u = load_unit(mat, t, k);
      build_index(mat, u, inv, pre);
      for (int c = 0; c < 4; ++c) {
        const int B = 1 << c, NW = 2 * B, per = 16 / B;
        const uint32_t mask = (1u << B) - 1;
        for (int e = threadIdx.x; e < u.n[c]; e += kThreads) {
          const int p = inv[u.base[c] + e];
          const int jl = p >> mat.logR, r = p & (mat.R - 1);
          const size_t g = (size_t)u.start[c] + e;
          const uint32_t* wv = (const uint32_t*)mat.codes[c] + g * NW;
          const float s = (float)__builtin_bit_cast(_Float16, mat.scales[c][g]);
          float* dst = W + ((size_t)t * mat.R + r) * mat.K + (size_t)(u.j0 + jl) * 64;
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
      }
      __syncthreads();
    }
  }
}

vbq_status make_dev_matrix(const vbq_desc* d, const void* blob, DevMatrix* m) {
  if (!d || !blob) return VBQ_ERR_NULL;
  vbq_status st = vbq_desc_check(d);
  if (st != VBQ_OK) return st;
  if ((uintptr_t)blob % 256 != 0) return VBQ_ERR_BUFFER;
  const uint8_t* b = (const uint8_t*)blob;
  m->units = (const uint32_t*)(b + d->section_off[VBQ_SEC_UNITS]);
  m->wmap = (const uint64_t*)(b + d->section_off[VBQ_SEC_WMAP]);
  for (int c = 0; c < 4; ++c) {
    m->codes[c] = b + d->section_off[VBQ_SEC_CODES0 + c];
    m->scales[c] = (const uint16_t*)(b + d->section_off[VBQ_SEC_SCALES0 + c]);
    m->n_entries[c] = (uint32_t)d->n_entries[c];
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

// Largest sub-chunk (group columns staged at once) that fits the LDS budget,
// keeping sub-chunk boundaries on width-map word boundaries (SC*R % 64 == 0).
int choose_sc(int R, int C, int MT) {
  const int step = R >= 64 ? 1 : 64 / R;
  for (int sc = C; sc >= 1; --sc) {
    if (sc != C && sc % step) continue;
    if (lds_plan(R, C, MT, sc).total <= 64 * 1024) return sc;
  }
  for (int sc = C; sc >= 1; --sc) {
    if (sc != C && sc % step) continue;
    if (lds_plan(R, C, MT, sc).total <= kLdsLimit) return sc;
  }
  return 0;
}

template <int MT>
vbq_status launch_mv(const DevMatrix& m, const void* x, int64_t ldx, int M, float* y, int64_t ldy, hipStream_t s) {
  MvArgs a;
  a.m = m;
  a.x = (const uint16_t*)x;
  a.y = y;
  a.ldx = ldx;
  a.ldy = ldy;
  a.M = M;
  a.SC = choose_sc(m.R, m.C, MT);
  if (a.SC <= 0) return VBQ_ERR_UNSUPPORTED;
  const int lds = lds_plan(m.R, m.C, MT, a.SC).total;
  static bool attr_set = false;  // raise the dynamic LDS limit once per process
  if (!attr_set) {
    if (hipFuncSetAttribute((const void*)vbq_mv_kernel<MT>, hipFuncAttributeMaxDynamicSharedMemorySize, kLdsLimit) !=
        hipSuccess)
      return VBQ_ERR_HIP;
    attr_set = true;
  }
  hipLaunchKernelGGL(vbq_mv_kernel<MT>, dim3((unsigned)m.T), dim3(kThreads), lds, s, a);
  return hipGetLastError() == hipSuccess ? VBQ_OK : VBQ_ERR_HIP;
}

}  // namespace

extern "C" {

vbq_status vbq_gemv(const vbq_desc* desc, const void* blob_dev, const void* x_dev, float* y_dev, void* stream) {
  if (!x_dev || !y_dev) return VBQ_ERR_NULL;
  DevMatrix m;
  vbq_status st = make_dev_matrix(desc, blob_dev, &m);
  if (st != VBQ_OK) return st;
  if ((uintptr_t)x_dev % 16 || (uintptr_t)y_dev % 4) return VBQ_ERR_BUFFER;
  return launch_mv<1>(m, x_dev, desc->K, 1, y_dev, desc->N, (hipStream_t)stream);
}

vbq_status vbq_gemm_small(const vbq_desc* desc, const void* blob_dev, int64_t M, const void* X_dev, int64_t ldx,
                          float* Y_dev, int64_t ldy, void* stream) {
  if (M < 0 || M > VBQ_MAX_M) return VBQ_ERR_SHAPE;
  DevMatrix m;
  vbq_status st = make_dev_matrix(desc, blob_dev, &m);
  if (st != VBQ_OK) return st;
  if (M == 0) return VBQ_OK;
  if (!X_dev || !Y_dev) return VBQ_ERR_NULL;
  if (ldx < desc->K || ldx % 8 || ldy < desc->N) return VBQ_ERR_SHAPE;
  if ((uintptr_t)X_dev % 16 || (uintptr_t)Y_dev % 4) return VBQ_ERR_BUFFER;
  hipStream_t s = (hipStream_t)stream;
  const int Mi = (int)M;
  if (Mi == 1) return launch_mv<1>(m, X_dev, ldx, 1, Y_dev, ldy, s);
  if (Mi == 2) return launch_mv<2>(m, X_dev, ldx, 2, Y_dev, ldy, s);
  if (Mi <= 4) return launch_mv<4>(m, X_dev, ldx, Mi, Y_dev, ldy, s);
  if (Mi <= 8) return launch_mv<8>(m, X_dev, ldx, Mi, Y_dev, ldy, s);
  return launch_mv<16>(m, X_dev, ldx, Mi, Y_dev, ldy, s);
}

vbq_status vbq_dequant(const vbq_desc* desc, const void* blob_dev, float* W_dev, void* stream) {
  if (!W_dev) return VBQ_ERR_NULL;
  DevMatrix m;
  vbq_status st = make_dev_matrix(desc, blob_dev, &m);
  if (st != VBQ_OK) return st;
  if ((uintptr_t)W_dev % 4) return VBQ_ERR_BUFFER;
  const int lds = align16(m.R * m.C * 2) + align16(4 * (kMaxWords + 1) * 2);
  hipLaunchKernelGGL(vbq_dequant_kernel, dim3((unsigned)m.T), dim3(kThreads), lds, (hipStream_t)stream, m, W_dev);
  return hipGetLastError() == hipSuccess ? VBQ_OK : VBQ_ERR_HIP;
}

}  // extern "C"
