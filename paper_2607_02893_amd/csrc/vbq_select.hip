// Differentiable bit selection on gfx950 (MI355X): the forward pass of the
// selection path (paper section 3.2, Algorithm 1) and the gradient of its
// logit step (section 3.3); the gradient kernel is described where it is
// defined.
//
// For every group g of 64 contiguous weights the forward kernel forms the four
// candidate reconstructions w_hat^(b), b in {1, 2, 4, 8} (section 3.1: Eq. (1)
// for b >= 2, sign times absmean for b = 1), the Gumbel-Softmax weights
// pi_g = softmax((l_g + e_g) / tau), and the soft weight
// w_soft = sum_k pi_{g,k} w_hat^(B_k); optionally also pi, the hardened width
// B[argmax_k l_{g,k}] and the expected bit cost bbar = mean_g sum_k pi_{g,k} B_k.
//
// The work is elementwise over a flat array of groups, so it is bound by HBM
// traffic (read W, write w_soft: 8 bytes per weight), not by arithmetic:
//   * one wave64 owns a slab of 64 consecutive groups (16 KiB of W) per step,
//     loaded with coalesced 16-byte buffer loads (the slab's buffer resource
//     ends at the last group, so a ragged last slab reads zeros and its
//     stores are dropped) and transposed through LDS so that each lane holds
//     one whole group;
//   * a lane computes its group's statistics in the order the quantizer
//     defines them: max|w| in fp32 (exact), the 1-bit absmean as the
//     sequential double sum / 64, each scale rounded once to fp16 from double
//     (via a round-to-odd float, which makes the two roundings one);
//   * round(w/s) is taken as rint(w * rcp(s)); the estimate is within 5e-5 of
//     w/s, so whenever it is farther than 2^-12 from a half-integer it is
//     exact, and otherwise (rare) the wave compares w with the exact midpoint
//     (q +- 1/2) * s, which is representable in fp32 (9-bit times 11-bit
//     significands), and applies round-half-to-even;
//   * pi_{g,k} * s_k is folded once per group, so each weight costs one FMA
//     per candidate in the mix;
//   * the next slab's loads are issued before the current slab's arithmetic;
//   * the results go back through LDS and out as coalesced 16-byte stores;
//   * the bulk loads and stores carry the non-temporal hint, and the grid is
//     2048 one-wave blocks (eight per CU), which measured fastest.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/vbq.h"

vbq_status vbq_detail_hip_status(hipError_t e);

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kGroupsPerSlab = 64;  // one group per lane
constexpr int kRowFloats = 68;      // LDS row of one group: 64 weights + 4 floats of padding
constexpr int kMaxBlocks = 2048;    // one wave per block; eight resident blocks per CU on 256 CUs
constexpr int kGradBlocks = 2048;   // the gradient's blocks: one tile + a 2 KiB table, eight resident per CU
constexpr int kBbarThreads = 256;
constexpr float kMinTau = 1.17549435e-38f;  // the smallest normal float: a subnormal tau may be flushed to 0
constexpr uint32_t kRsrcFlags = 0x00020000;
// Cache policy of the bulk weight loads and w_soft stores: non-temporal (each
// byte is touched once).  Measured on the 131M-class step: 221 us with the
// hint, 253 us without; the hint on the small per-group arrays costs time.
constexpr int kNonTemporal = 2;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, (int)kRsrcFlags);
}

__device__ __forceinline__ void lds_store_u32x4(uint32_t addr, u32x4 v) {
  *(__attribute__((address_space(3))) u32x4*)(size_t)addr = v;
}
__device__ __forceinline__ u32x4 lds_u32x4(uint32_t addr) {
  return *(__attribute__((address_space(3))) u32x4*)(size_t)addr;
}

// fp16 value nearest to d >= 0 (round to nearest even), with one rounding:
// d is first rounded to float by round-to-odd, which keeps enough bits (24 >=
// 11 + 2) for the float -> fp16 conversion to round as if from d itself.
__device__ __forceinline__ float fp16_from_double(double d) {
  float f = (float)d;
  if ((double)f != d) {
    uint32_t b = __builtin_bit_cast(uint32_t, f);
    if ((double)f > d) b -= 1u;  // the float below d (d > 0 here)
    f = __builtin_bit_cast(float, b | 1u);
  }
  return (float)(_Float16)f;
}

// Components of a 4 x 32-bit vector are reinterpreted with __uint_as_float /
// __float_as_uint: __builtin_bit_cast applied to a vector component (t.y)
// reads the wrong component with this compiler.

struct Cand {   // one candidate width of one group
  float s;      // stored scale (an fp16 value), 0 for an all-zero group
  float r;      // approximate 1/s (0 when s == 0)
  float c;      // pi_k * s
  float qmax;
};

// Exact round-half-to-even of w/s given an estimate q0 within one of it.
__device__ __forceinline__ float exact_rne(float w, float q0, float s) {
  const float p = q0 * s;                          // exact: 9-bit times 11-bit significand
  const float sg = w > p ? 1.0f : (w < p ? -1.0f : 0.0f);
  const float b = __builtin_fmaf(0.5f, sg, q0) * s;  // midpoint toward w, exact
  const bool beyond = sg > 0.0f ? (w > b) : (w < b);
  const bool odd = (((int)q0) & 1) != 0;
  const bool step = beyond || (w == b && odd);
  return step ? q0 + sg : q0;
}

// The four candidates' scales of one group (section 3.1), from the group's
// 64 weights in the lane's LDS row: max|w| in fp32 (exact), the 1-bit absmean
// as the sequential double sum / 64, every scale rounded once to fp16.
struct Scales {
  float s1;
  Cand c2, c4, c8;
};

__device__ __forceinline__ Scales group_scales(uint32_t row_addr) {
  float amax = 0.0f;
  double asum = 0.0;
#pragma unroll 4
  for (int j = 0; j < 16; ++j) {
    const u32x4 t = lds_u32x4(row_addr + 16u * j);
    const float f[4] = {__uint_as_float(t.x), __uint_as_float(t.y), __uint_as_float(t.z), __uint_as_float(t.w)};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      amax = __builtin_fmaxf(amax, __builtin_fabsf(f[i]));
      asum += (double)__builtin_fabsf(f[i]);  // sequential, weight 0 to 63
    }
  }
  Scales sc;
  sc.s1 = fp16_from_double(asum * (1.0 / 64.0));
  sc.c2.s = fp16_from_double((double)amax);
  sc.c4.s = fp16_from_double((double)amax / 7.0);
  sc.c8.s = fp16_from_double((double)amax / 127.0);
  sc.c2.qmax = 1.0f;
  sc.c4.qmax = 7.0f;
  sc.c8.qmax = 127.0f;
  sc.c2.r = sc.c2.s > 0.0f ? __builtin_amdgcn_rcpf(sc.c2.s) : 0.0f;
  sc.c4.r = sc.c4.s > 0.0f ? __builtin_amdgcn_rcpf(sc.c4.s) : 0.0f;
  sc.c8.r = sc.c8.s > 0.0f ? __builtin_amdgcn_rcpf(sc.c8.s) : 0.0f;
  return sc;
}

// Levels q = clip(round(x/s), -qmax, qmax) of the 2-, 4- and 8-bit candidates
// (Eq. (1)), round-half-to-even exactly: rint(x * rcp(s)) is within 5e-5 of
// x/s, so it is exact unless within 2^-12 of a half-integer; then the wave
// takes the midpoint comparison for every lane.
__device__ __forceinline__ void levels(float x, const Scales& sc, float& q2, float& q4, float& q8) {
  constexpr float kNear = 0.5f - 1.0f / 4096.0f;
  const float t2 = x * sc.c2.r, t4 = x * sc.c4.r, t8 = x * sc.c8.r;
  q2 = __builtin_rintf(t2);
  q4 = __builtin_rintf(t4);
  q8 = __builtin_rintf(t8);
  const bool near = __builtin_fabsf(t2 - q2) > kNear || __builtin_fabsf(t4 - q4) > kNear ||
                    __builtin_fabsf(t8 - q8) > kNear;
  if (__builtin_amdgcn_ballot_w64(near)) {
    q2 = exact_rne(x, q2, sc.c2.s);
    q4 = exact_rne(x, q4, sc.c4.s);
    q8 = exact_rne(x, q8, sc.c8.s);
  }
  q2 = __builtin_amdgcn_fmed3f(q2, -sc.c2.qmax, sc.c2.qmax);
  q4 = __builtin_amdgcn_fmed3f(q4, -sc.c4.qmax, sc.c4.qmax);
  q8 = __builtin_amdgcn_fmed3f(q8, -sc.c8.qmax, sc.c8.qmax);
}

// LDS byte addresses of one lane: in the coalesced phase load j covers groups
// 4j .. 4j+3 and lane l holds the 4 floats at (group 4j + l/16, weight
// 4*(l%16)); in the lane-per-group phase lane l owns row l.
struct TileAddr {
  uint32_t co[16];
  uint32_t row;
};

__device__ __forceinline__ TileAddr tile_addr(uint32_t base, uint32_t lane) {
  TileAddr t;
#pragma unroll
  for (int j = 0; j < 16; ++j) t.co[j] = base + 4u * ((4u * j + (lane >> 4)) * kRowFloats + 4u * (lane & 15u));
  t.row = base + 4u * lane * kRowFloats;
  return t;
}

struct QatArgs {
  const float* W;
  const float* logits;
  const float* noise;  // may be null
  void* w_soft;        // float, or bf16 with kBf16
  float* pi;           // may be null
  uint8_t* hard;       // may be null
  double* partial;     // per-block sums of sum_k pi_k B_k, or null
  float tau;
  int64_t n_groups;
  int64_t n_slabs;
};

// Two fp32 values as a bf16 pair, each rounded to nearest even (one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t bf16_pair(float lo, float hi) {
  const bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

template <bool kBf16>
__global__ __launch_bounds__(64) void vbq_qat_forward_kernel(QatArgs a) {
  __shared__ __attribute__((aligned(16))) float tile[kGroupsPerSlab * kRowFloats];
  const uint32_t lane = threadIdx.x;
  const uint32_t base = (uint32_t)(size_t)(__attribute__((address_space(3))) float*)tile;
  const TileAddr ta = tile_addr(base, lane);
  const uint32_t* co_addr = ta.co;
  const uint32_t row_addr = ta.row;

  double eb_sum = 0.0;
  int64_t slab = blockIdx.x;
  const int64_t stride = gridDim.x;
  u32x4 v[16];
  u32x4 lg = {0, 0, 0, 0}, ns = {0, 0, 0, 0};
  auto load_slab = [&](int64_t sl) {
    const int64_t g0 = sl * kGroupsPerSlab;
    const int64_t left = a.n_groups - g0;
    const uint32_t ng = (uint32_t)(left < kGroupsPerSlab ? left : kGroupsPerSlab);
    const __amdgpu_buffer_rsrc_t rw = rsrc(a.W + g0 * 64, ng * 256u);
#pragma unroll
    for (int j = 0; j < 16; ++j) v[j] = __builtin_amdgcn_raw_buffer_load_b128(rw, (int)(j * 1024 + lane * 16), 0, kNonTemporal);
    lg = __builtin_amdgcn_raw_buffer_load_b128(rsrc(a.logits + g0 * 4, ng * 16u), (int)(lane * 16), 0, 0);
    if (a.noise) ns = __builtin_amdgcn_raw_buffer_load_b128(rsrc(a.noise + g0 * 4, ng * 16u), (int)(lane * 16), 0, 0);
  };
  if (slab < a.n_slabs) load_slab(slab);

  for (; slab < a.n_slabs; slab += stride) {
    const int64_t g0 = slab * kGroupsPerSlab;
    const int64_t left = a.n_groups - g0;
    const uint32_t ng = (uint32_t)(left < kGroupsPerSlab ? left : kGroupsPerSlab);

    // ---- transpose the slab through LDS: row `lane` holds group g0 + lane
#pragma unroll
    for (int j = 0; j < 16; ++j) lds_store_u32x4(co_addr[j], v[j]);
    __syncthreads();
    const float l0 = __uint_as_float(lg.x), l1 = __uint_as_float(lg.y);
    const float l2 = __uint_as_float(lg.z), l3 = __uint_as_float(lg.w);
    const float e0 = __uint_as_float(ns.x), e1 = __uint_as_float(ns.y);
    const float e2 = __uint_as_float(ns.z), e3 = __uint_as_float(ns.w);
    // ---- the next slab's loads overlap this slab's arithmetic
    if (slab + stride < a.n_slabs) load_slab(slab + stride);

    // ---- group statistics and scales (section 3.1), streaming the lane's row
    const Scales sc = group_scales(row_addr);
    const float s1 = sc.s1;
    Cand c2 = sc.c2, c4 = sc.c4, c8 = sc.c8;

    // ---- Gumbel-Softmax weights (section 3.2); the largest l + e is subtracted
    // before the division, so a small tau cannot overflow to inf - inf
    const float v0 = l0 + e0, v1 = l1 + e1, v2 = l2 + e2, v3 = l3 + e3;
    const float vm = __builtin_fmaxf(__builtin_fmaxf(v0, v1), __builtin_fmaxf(v2, v3));
    const float p0 = expf((v0 - vm) / a.tau), p1 = expf((v1 - vm) / a.tau), p2 = expf((v2 - vm) / a.tau),
                p3 = expf((v3 - vm) / a.tau);
    const float psum = (p0 + p1) + (p2 + p3);
    const float pi0 = p0 / psum, pi1 = p1 / psum, pi2 = p2 / psum, pi3 = p3 / psum;
    const float c1 = pi0 * s1;
    c2.c = pi1 * c2.s;
    c4.c = pi2 * c4.s;
    c8.c = pi3 * c8.s;
    const bool valid = lane < ng;
    if (valid) eb_sum += (double)(pi0 + 2.0f * pi1 + 4.0f * pi2 + 8.0f * pi3);
    if (a.pi) {
      const u32x4 pv = {__float_as_uint(pi0), __float_as_uint(pi1),
                        __float_as_uint(pi2), __float_as_uint(pi3)};
      __builtin_amdgcn_raw_buffer_store_b128(pv, rsrc(a.pi + g0 * 4, ng * 16u), (int)(lane * 16), 0, 0);
    }
    if (a.hard) {
      // Algorithm 1's result: the width of the largest logit (the first of equal maxima)
      int k = 0;
      float best = l0;
      if (l1 > best) { best = l1; k = 1; }
      if (l2 > best) { best = l2; k = 2; }
      if (l3 > best) { k = 3; }
      __builtin_amdgcn_raw_buffer_store_b8((uint8_t)(1u << k), rsrc(a.hard + g0, ng), (int)lane, 0, 0);
    }

    // ---- the mix, four weights at a time, in place in the lane's row
#pragma unroll 2
    for (int j = 0; j < 16; ++j) {
      const u32x4 t = lds_u32x4(row_addr + 16u * j);
      float f[4] = {__uint_as_float(t.x), __uint_as_float(t.y), __uint_as_float(t.z), __uint_as_float(t.w)};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float x = f[i];
        float q2, q4, q8;
        levels(x, sc, q2, q4, q8);
        float acc = x >= 0.0f ? c1 : -c1;  // sign(0) = +1 (also for -0.0)
        acc = __builtin_fmaf(c2.c, q2, acc);
        acc = __builtin_fmaf(c4.c, q4, acc);
        acc = __builtin_fmaf(c8.c, q8, acc);
        f[i] = acc;
      }
      const u32x4 o = {__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]), __float_as_uint(f[3])};
      lds_store_u32x4(row_addr + 16u * j, o);
    }

    // ---- out of LDS with coalesced stores (bf16: each float rounded to nearest even)
    __syncthreads();
    if constexpr (kBf16) {
      const __amdgpu_buffer_rsrc_t ro = rsrc((const uint16_t*)a.w_soft + g0 * 64, ng * 128u);
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const u32x4 t = lds_u32x4(co_addr[j]);
        const u32x2 o = {bf16_pair(__uint_as_float(t.x), __uint_as_float(t.y)),
                         bf16_pair(__uint_as_float(t.z), __uint_as_float(t.w))};
        __builtin_amdgcn_raw_buffer_store_b64(o, ro, (int)(j * 512 + lane * 8), 0, kNonTemporal);
      }
    } else {
      const __amdgpu_buffer_rsrc_t ro = rsrc((const float*)a.w_soft + g0 * 64, ng * 256u);
#pragma unroll
      for (int j = 0; j < 16; ++j)
        __builtin_amdgcn_raw_buffer_store_b128(lds_u32x4(co_addr[j]), ro, (int)(j * 1024 + lane * 16), 0, kNonTemporal);
    }
    __syncthreads();  // the next slab overwrites the tile
  }

  if (a.partial) {
    // fixed-order butterfly over the wave: the same grid gives the same sum
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) eb_sum += __shfl_xor(eb_sum, d, 64);
    if (lane == 0) a.partial[blockIdx.x] = eb_sum;
  }
}

struct GradArgs {
  const float* W;
  const float* grad;   // dL/dw_soft
  const float* pi;
  float* dlogits;
  float tau;
  float lambda;
  double n_bbar;       // the n of bbar
  int64_t n_groups;
  int64_t n_slabs;
};

// Sum of v over each row of 16 lanes, every lane of the row receiving it, in
// a fixed order (quad swaps, then the half-row and row mirrors).
constexpr int kDppQuadXor1 = 0xB1, kDppQuadXor2 = 0x4E, kDppRowHalfMirror = 0x141, kDppRowMirror = 0x140;

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __uint_as_float((uint32_t)__builtin_amdgcn_update_dpp(0, (int)__float_as_uint(v), CTRL, 0xf, 0xf, true));
}

__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_f32<kDppQuadXor1>(v);
  v += dpp_f32<kDppQuadXor2>(v);
  v += dpp_f32<kDppRowHalfMirror>(v);
  v += dpp_f32<kDppRowMirror>(v);
  return v;
}

// Logit step of Algorithm 1 (section 3.3): with the candidates held constant,
//   a_k = sum_i G_i w_hat^(B_k)_i + lambda B_k / n,
//   dL/dl_k = (pi_k / tau) (a_k - sum_j pi_j a_j).
// Same slab walk as the forward.  The weights go through the LDS tile only for
// the group statistics (lane per group, the quantizer's order); the scales go
// to a small per-group table, and the products run in the coalesced layout of
// the loads: lane l of load j holds weights and gradients 4(l%16) .. +3 of
// group 4j + l/16, so the gradients never pass through LDS.  The four sums of
// a group are reduced over its 16 lanes (fixed DPP order) and parked in the
// padding of the group's tile row, where the lane that owns the group picks
// them up.  The next slab's weights are loaded while this slab is worked on;
// its gradients are loaded at the slab's start (a second gradient buffer
// would cost the second wave per SIMD: 268 VGPRs, measured slower).
// sum_i G_i w_hat^(b)_i = s_b sum_i G_i q_i.
__global__ __launch_bounds__(64) void vbq_qat_grad_kernel(GradArgs a) {
  __shared__ __attribute__((aligned(16))) float tile[kGroupsPerSlab * kRowFloats];
  __shared__ __attribute__((aligned(16))) float consts[kGroupsPerSlab * 8];  // s1 s2 s4 s8 r2 r4 r8 -
  const uint32_t lane = threadIdx.x;
  const uint32_t base = (uint32_t)(size_t)(__attribute__((address_space(3))) float*)tile;
  const uint32_t cbase = (uint32_t)(size_t)(__attribute__((address_space(3))) float*)consts;
  const TileAddr ta = tile_addr(base, lane);
  const float pen1 = (float)((double)a.lambda * 1.0 / a.n_bbar), pen2 = (float)((double)a.lambda * 2.0 / a.n_bbar);
  const float pen4 = (float)((double)a.lambda * 4.0 / a.n_bbar), pen8 = (float)((double)a.lambda * 8.0 / a.n_bbar);
  const int64_t stride = gridDim.x;

  u32x4 v[16];
  auto load_slab = [&](int64_t sl) __attribute__((always_inline)) {
    const int64_t g0 = sl * kGroupsPerSlab;
    const int64_t left = a.n_groups - g0;
    const uint32_t ng = (uint32_t)(left < kGroupsPerSlab ? left : kGroupsPerSlab);
    const __amdgpu_buffer_rsrc_t rw = rsrc(a.W + g0 * 64, ng * 256u);
#pragma unroll
    for (int j = 0; j < 16; ++j) v[j] = __builtin_amdgcn_raw_buffer_load_b128(rw, (int)(j * 1024 + lane * 16), 0, kNonTemporal);
  };

  // one slab; its gradients are loaded at its start, coalesced, at the
  // weights' offsets
  auto step = [&](int64_t sl) __attribute__((always_inline)) {
    const int64_t g0 = sl * kGroupsPerSlab;
    const int64_t left = a.n_groups - g0;
    const uint32_t ng = (uint32_t)(left < kGroupsPerSlab ? left : kGroupsPerSlab);
#pragma unroll
    for (int j = 0; j < 16; ++j) lds_store_u32x4(ta.co[j], v[j]);
    __syncthreads();
    u32x4 gv[16];
    const __amdgpu_buffer_rsrc_t rg = rsrc(a.grad + g0 * 64, ng * 256u);
#pragma unroll
    for (int j = 0; j < 16; ++j) gv[j] = __builtin_amdgcn_raw_buffer_load_b128(rg, (int)(j * 1024 + lane * 16), 0, kNonTemporal);
    const u32x4 pv = __builtin_amdgcn_raw_buffer_load_b128(rsrc(a.pi + g0 * 4, ng * 16u), (int)(lane * 16), 0, 0);
    if (sl + stride < a.n_slabs) load_slab(sl + stride);

    // ---- scales of this lane's group, into the per-group table
    const Scales own = group_scales(ta.row);
    lds_store_u32x4(cbase + 32u * lane, u32x4{__float_as_uint(own.s1), __float_as_uint(own.c2.s),
                                              __float_as_uint(own.c4.s), __float_as_uint(own.c8.s)});
    lds_store_u32x4(cbase + 32u * lane + 16u, u32x4{__float_as_uint(own.c2.r), __float_as_uint(own.c4.r),
                                                    __float_as_uint(own.c8.r), 0u});
    __syncthreads();

    // ---- products in the coalesced layout; sums of group 4j + lane/16 over its 16 lanes
    // (fully unrolled: gv[j] must stay in registers)
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const uint32_t grp = 4u * j + (lane >> 4);
      const u32x4 c0 = lds_u32x4(cbase + 32u * grp), c1 = lds_u32x4(cbase + 32u * grp + 16u);
      Scales sc;
      sc.s1 = __uint_as_float(c0.x);
      sc.c2.s = __uint_as_float(c0.y);
      sc.c4.s = __uint_as_float(c0.z);
      sc.c8.s = __uint_as_float(c0.w);
      sc.c2.r = __uint_as_float(c1.x);
      sc.c4.r = __uint_as_float(c1.y);
      sc.c8.r = __uint_as_float(c1.z);
      sc.c2.qmax = 1.0f;
      sc.c4.qmax = 7.0f;
      sc.c8.qmax = 127.0f;
      const u32x4 t = lds_u32x4(ta.co[j]);
      const float f[4] = {__uint_as_float(t.x), __uint_as_float(t.y), __uint_as_float(t.z), __uint_as_float(t.w)};
      const float gr[4] = {__uint_as_float(gv[j].x), __uint_as_float(gv[j].y), __uint_as_float(gv[j].z),
                           __uint_as_float(gv[j].w)};
      float d1 = 0.0f, d2 = 0.0f, d4 = 0.0f, d8 = 0.0f;  // sum G q per candidate, this lane's 4 weights
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float q2, q4, q8;
        levels(f[i], sc, q2, q4, q8);
        d1 += f[i] >= 0.0f ? gr[i] : -gr[i];  // sign(0) = +1
        d2 = __builtin_fmaf(gr[i], q2, d2);
        d4 = __builtin_fmaf(gr[i], q4, d4);
        d8 = __builtin_fmaf(gr[i], q8, d8);
      }
      d1 = row16_sum(d1);
      d2 = row16_sum(d2);
      d4 = row16_sum(d4);
      d8 = row16_sum(d8);
      // the row's first lane parks the group's sums in the padding of the group's tile row
      if ((lane & 15u) == 0)
        lds_store_u32x4(base + 4u * (grp * kRowFloats + 64u),
                        u32x4{__float_as_uint(d1), __float_as_uint(d2), __float_as_uint(d4), __float_as_uint(d8)});
    }
    __syncthreads();

    // ---- lane per group: the logit gradient of group g0 + lane
    const u32x4 dv = lds_u32x4(ta.row + 256u);
    const float a1 = __builtin_fmaf(own.s1, __uint_as_float(dv.x), pen1);
    const float a2 = __builtin_fmaf(own.c2.s, __uint_as_float(dv.y), pen2);
    const float a4 = __builtin_fmaf(own.c4.s, __uint_as_float(dv.z), pen4);
    const float a8 = __builtin_fmaf(own.c8.s, __uint_as_float(dv.w), pen8);
    const float p0 = __uint_as_float(pv.x), p1 = __uint_as_float(pv.y), p2 = __uint_as_float(pv.z),
                p3 = __uint_as_float(pv.w);
    const float mean = (p0 * a1 + p1 * a2) + (p2 * a4 + p3 * a8);
    const u32x4 out = {__float_as_uint(p0 / a.tau * (a1 - mean)), __float_as_uint(p1 / a.tau * (a2 - mean)),
                       __float_as_uint(p2 / a.tau * (a4 - mean)), __float_as_uint(p3 / a.tau * (a8 - mean))};
    __builtin_amdgcn_raw_buffer_store_b128(out, rsrc(a.dlogits + g0 * 4, ng * 16u), (int)(lane * 16), 0, 0);
    __syncthreads();  // the next slab overwrites the tile and the table
  };

  int64_t slab = blockIdx.x;
  if (slab < a.n_slabs) load_slab(slab);
  for (; slab < a.n_slabs; slab += stride) step(slab);
}

// bbar = (sum of the per-block sums) / n_groups, summed in a fixed order.
__global__ __launch_bounds__(kBbarThreads) void vbq_qat_bbar_kernel(const double* partial, int n, double n_groups,
                                                                    double* bbar) {
  __shared__ double red[kBbarThreads];
  double s = 0.0;
  for (int i = threadIdx.x; i < n; i += kBbarThreads) s += partial[i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int h = kBbarThreads / 2; h >= 1; h >>= 1) {
    if ((int)threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) *bbar = red[0] / n_groups;
}

int64_t qat_blocks(int64_t n_groups) {
  const int64_t slabs = (n_groups + kGroupsPerSlab - 1) / kGroupsPerSlab;
  return slabs < kMaxBlocks ? slabs : kMaxBlocks;
}

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p % a) == 0; }

}  // namespace

extern "C" {

vbq_status vbq_qat_workspace_size(int64_t n_groups, size_t* bytes) {
  if (!bytes) return VBQ_ERR_NULL;
  if (n_groups < 0 || n_groups > VBQ_QAT_MAX_GROUPS) return VBQ_ERR_SHAPE;
  *bytes = (size_t)qat_blocks(n_groups) * sizeof(double);
  return VBQ_OK;
}

vbq_status vbq_qat_forward(int64_t n_groups, const float* W_dev, const float* logits_dev, const float* noise_dev,
                           float tau, uint32_t flags, void* w_soft_dev, float* pi_dev, uint8_t* hard_bits_dev,
                           double* bbar_dev, void* workspace_dev, size_t workspace_bytes, void* stream) {
  if (n_groups < 0 || n_groups > VBQ_QAT_MAX_GROUPS) return VBQ_ERR_SHAPE;
  if (!(tau == tau) || tau == __builtin_inff() || tau == -__builtin_inff()) return VBQ_ERR_NONFINITE;
  if (!(tau >= kMinTau)) return VBQ_ERR_UNSUPPORTED;
  if (flags & ~VBQ_QAT_WSOFT_BF16) return VBQ_ERR_UNSUPPORTED;
  if (n_groups == 0) return VBQ_OK;
  if (!W_dev || !logits_dev || !w_soft_dev) return VBQ_ERR_NULL;
  if (!aligned(W_dev, 16) || !aligned(logits_dev, 16) || !aligned(w_soft_dev, 16) ||
      (noise_dev && !aligned(noise_dev, 16)) || (pi_dev && !aligned(pi_dev, 16)))
    return VBQ_ERR_BUFFER;
  const int64_t blocks = qat_blocks(n_groups);
  if (bbar_dev) {
    if (!workspace_dev) return VBQ_ERR_NULL;
    if (!aligned(bbar_dev, 8) || !aligned(workspace_dev, 8) || workspace_bytes < (size_t)blocks * sizeof(double))
      return VBQ_ERR_BUFFER;
  }
  hipStream_t s = (hipStream_t)stream;
  QatArgs a;
  a.W = W_dev;
  a.logits = logits_dev;
  a.noise = noise_dev;
  a.w_soft = w_soft_dev;
  a.pi = pi_dev;
  a.hard = hard_bits_dev;
  a.partial = bbar_dev ? (double*)workspace_dev : nullptr;
  a.tau = tau;
  a.n_groups = n_groups;
  a.n_slabs = (n_groups + kGroupsPerSlab - 1) / kGroupsPerSlab;
  void* args[] = {&a};
  const void* kernel = (flags & VBQ_QAT_WSOFT_BF16) ? (const void*)vbq_qat_forward_kernel<true>
                                                    : (const void*)vbq_qat_forward_kernel<false>;
  vbq_status st = vbq_detail_hip_status(hipLaunchKernel(kernel, dim3((unsigned)blocks), dim3(64), args, 0, s));
  if (st != VBQ_OK || !bbar_dev) return st;
  const double* part = (const double*)workspace_dev;
  int n = (int)blocks;
  double ngd = (double)n_groups;
  void* args2[] = {&part, &n, &ngd, &bbar_dev};
  return vbq_detail_hip_status(
      hipLaunchKernel((const void*)vbq_qat_bbar_kernel, dim3(1), dim3(kBbarThreads), args2, 0, s));
}

vbq_status vbq_qat_logit_grad(int64_t n_groups, const float* W_dev, const float* grad_dev, const float* pi_dev,
                              float tau, float lambda, int64_t n_bbar, float* dlogits_dev, void* stream) {
  if (n_groups < 0 || n_groups > VBQ_QAT_MAX_GROUPS) return VBQ_ERR_SHAPE;
  if (!(tau == tau) || tau == __builtin_inff() || tau == -__builtin_inff()) return VBQ_ERR_NONFINITE;
  if (!(lambda == lambda) || lambda == __builtin_inff() || lambda == -__builtin_inff()) return VBQ_ERR_NONFINITE;
  if (!(tau >= kMinTau)) return VBQ_ERR_UNSUPPORTED;
  if (n_bbar < 1) return VBQ_ERR_SHAPE;
  if (n_groups == 0) return VBQ_OK;
  if (!W_dev || !grad_dev || !pi_dev || !dlogits_dev) return VBQ_ERR_NULL;
  if (!aligned(W_dev, 16) || !aligned(grad_dev, 16) || !aligned(pi_dev, 16) || !aligned(dlogits_dev, 16))
    return VBQ_ERR_BUFFER;
  GradArgs a;
  a.W = W_dev;
  a.grad = grad_dev;
  a.pi = pi_dev;
  a.dlogits = dlogits_dev;
  a.tau = tau;
  a.lambda = lambda;
  a.n_bbar = (double)n_bbar;
  a.n_groups = n_groups;
  a.n_slabs = (n_groups + kGroupsPerSlab - 1) / kGroupsPerSlab;
  void* args[] = {&a};
  const int64_t blocks = a.n_slabs < kGradBlocks ? a.n_slabs : kGradBlocks;
  return vbq_detail_hip_status(hipLaunchKernel((const void*)vbq_qat_grad_kernel, dim3((unsigned)blocks), dim3(64),
                                               args, 0, (hipStream_t)stream));
}

}  // extern "C"
