/*
 * vbq.h -- C ABI of libvbq: packed variable-bit-width weights (VBQ) and the
 * fused dequantize-and-multiply used by autoregressive decode, for AMD
 * Instinct MI355X (gfx950).
 *
 * Method (arxiv 2607.02893, "Variable Bit-width Quantization"):
 *   - A weight matrix W[N][K] is cut into contiguous groups of G = 64 weights
 *     along K.  Group g has its own bit-width b_g in {1,2,4,8} and its own
 *     scale s_g (paper section 3.1).
 *   - b >= 2 (paper Eq. (1)): symmetric absmax,
 *       s = max|w| / (2^(b-1)-1),  q = clip(round(w/s), -(2^(b-1)-1), 2^(b-1)-1),
 *       w_hat = s*q.
 *   - b = 1 (paper section 3.1, text after Eq. (1)): w_hat = sign(w) * mean|w|.
 *   - Decode streams the packed low-bit codes, expands them in registers with
 *     the group scale and accumulates the matrix-vector product; the
 *     full-precision matrix is never materialised (paper section 6, "Fused
 *     kernels over packed weights").
 *   - Training chooses the widths (paper section 3.2, Algorithm 1): each group
 *     mixes its four candidate reconstructions with Gumbel-Softmax weights;
 *     vbq_qat_forward computes that mix (last part of this header).
 *
 * Readings fixed by this library where the paper is silent:
 *   - round() is round-half-to-even; the codes are computed against the scale
 *     AFTER it has been rounded to fp16 (so quantize(dequantize(q)) == q).
 *   - scales are IEEE fp16, computed in double and rounded once (RNE).
 *   - sign(0) = +1 for the 1-bit rule (also for -0.0).
 *   - the 1-bit absmean is the sequential double sum over the 64 weights / 64.
 *   - an all-zero group at b >= 2 has s = 0 and q = 0.
 *   - the level set of width b >= 2 is {-(2^(b-1)-1) .. 2^(b-1)-1}; the code
 *     for -2^(b-1) is never produced and is rejected by vbq_pack_codes.
 *   - K must be a multiple of 64 (a partial group would change the 1-bit mean).
 *   - products are accumulated in fp32; y is fp32.
 *
 * ---------------------------------------------------------------------------
 * Packed layout, version 1 (the paper leaves the storage format open; this is
 * the format every entry point below reads or writes)
 * ---------------------------------------------------------------------------
 *   G   = K/64 group columns.  Class c = log2(b): 0:1-bit 1:2-bit 2:4-bit 3:8-bit.
 *   R   = tile_rows (power of two in [16,256]); T = ceil(N/R) row tiles.
 *   C   = chunk_groups (1..128, R*C <= 8192); U = ceil(G/C) column chunks.
 *   Unit (t,k), u = t*U + k, covers rows [tR, min(N,tR+R)) and group columns
 *   [kC, min(G,kC+C)).  Inside a unit, position p = (j-kC)*R + (r-tR) for
 *   group column j and row r ("column-major"; the stride is R even in the last,
 *   ragged tile, whose missing rows are padding positions).
 *   Codes are offset-binary: u = q + 2^(b-1) for b >= 2, u = (q+1)/2 for b = 1.
 *
 *   Sections (each starts at a 256-byte aligned offset from the blob start):
 *   [0] unit table  uint32[n_units+1][8]: row u = {e0,e1,e2,e3, wmap_word, 0,0,0}
 *                   e_c = index of unit u's first class-c entry in section c;
 *                   wmap_word = index of unit u's first 64-bit word in [1].
 *                   Row n_units holds the totals.
 *   [1] wmap        uint64 words.  Unit u owns 2*W_u words, W_u = ceil(C_k*R/64):
 *                   W_u words of plane 0 (class bit 0) then W_u of plane 1
 *                   (class bit 1); position p is bit p%64 of word p/64.
 *                   Padding positions and the tail of the last word are 0.
 *   [2+c] codes[c]  class-c entries (groups of width 2^c), ordered by unit,
 *                   then by position p.  An entry is 8*b bytes = 2b little-
 *                   endian uint32 words.  Weight pair i (weights 2i, 2i+1 of
 *                   the group, i = 0..31) lives in word i / (16/b), field
 *                   f = i % (16/b): the code of weight 2i in bits
 *                   [f*b, f*b+b) and the code of weight 2i+1 in bits
 *                   [16+f*b, 16+f*b+b).
 *   [6+c] scales[c] IEEE fp16 bit patterns (uint16), one per class-c entry,
 *                   same order as codes[c].
 *
 * Conventions for every call:
 *   - The caller owns every buffer.  No entry point allocates device memory or
 *     keeps global state; calls on different streams are independent.
 *   - vbq_pack* run synchronously on the host.  Device entry points enqueue
 *     work on the given stream and return; errors detected before the launch
 *     are returned, a failed launch returns VBQ_ERR_HIP.
 *   - Device pointers must be 16-byte aligned; x / X are contiguous fp16.
 *   - Nothing throws across this interface.
 *   - The library reads no environment variables: every option of a device
 *     call is a bit of vbq_desc.flags (VBQ_Y_F16, VBQ_ONE_WAVE_PER_UNIT below),
 *     read once per call.
 */
#ifndef VBQ_H
#define VBQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum vbq_status {
  VBQ_OK = 0,
  VBQ_ERR_NULL = 1,        /* a required pointer is NULL                      */
  VBQ_ERR_SHAPE = 2,       /* N < 1, K < 64, K % 64 != 0, M out of range, ... */
  VBQ_ERR_BITS = 3,        /* a bit-width outside {1,2,4,8}                   */
  VBQ_ERR_CODE_RANGE = 4,  /* a code outside its width's level set            */
  VBQ_ERR_NONFINITE = 5,   /* NaN or Inf in weights, or a non-finite scale    */
  VBQ_ERR_SCALE_RANGE = 6, /* a scale that rounds to Inf in fp16, or < 0      */
  VBQ_ERR_BUFFER = 7,      /* buffer too small or misaligned                  */
  VBQ_ERR_DESC = 8,        /* descriptor magic / version / shape mismatch     */
  VBQ_ERR_HIP = 9,         /* the HIP runtime reported an error               */
  VBQ_ERR_UNSUPPORTED = 10 /* option outside the supported range              */
} vbq_status;

#define VBQ_MAGIC 0x31514256u /* "VBQ1" little-endian */
#define VBQ_LAYOUT_VERSION 1u
#define VBQ_GROUP 64
#define VBQ_NSECTIONS 10
#define VBQ_MAX_M 16

/* vbq_desc.flags: options of the device calls that take the descriptor
 * (vbq_gemv, vbq_gemv_rows, vbq_gemm_small, and the matrices of a step plan),
 * read on every call.  The packers write 0; set bits on a copy of the
 * descriptor to choose them.  Other bits give VBQ_ERR_UNSUPPORTED.
 *   VBQ_Y_F16             y / Y is written as IEEE fp16 (each fp32 result
 *                         rounded to nearest even): at most 2^-11 relative
 *                         error added for |y| in [2^-14, 65504], at most 2^-25
 *                         absolute below that, +-inf from 65520 up.  y / Y must
 *                         then be 2-byte aligned (4 bytes for float).  Ignored
 *                         by vbq_dequant.
 *   VBQ_ONE_WAVE_PER_UNIT the one- and two-row products use one wave per unit
 *                         even where the library would use two (small
 *                         mixed-width matrices).  Results agree within the
 *                         output tolerance, bitwise where both take whole
 *                         units; it exists so both kernels can be compared on
 *                         the same inputs. */
#define VBQ_Y_F16 1u
#define VBQ_ONE_WAVE_PER_UNIT 2u
#define VBQ_CALL_FLAGS (VBQ_Y_F16 | VBQ_ONE_WAVE_PER_UNIT)

/* Section indices in vbq_desc.section_off / section_len. */
enum { VBQ_SEC_UNITS = 0, VBQ_SEC_WMAP = 1, VBQ_SEC_CODES0 = 2, VBQ_SEC_SCALES0 = 6 };

/* Host-side description of one packed matrix (plain old data). */
typedef struct vbq_desc {
  uint32_t magic;        /* VBQ_MAGIC                                  */
  uint32_t version;      /* VBQ_LAYOUT_VERSION                         */
  int64_t N, K;          /* rows (outputs) and columns (inputs)        */
  int32_t group;         /* always 64                                  */
  int32_t tile_rows;     /* R                                          */
  int32_t chunk_groups;  /* C                                          */
  int32_t reserved0;
  int64_t n_tiles, n_chunks, n_units;
  int64_t n_entries[4];  /* number of groups of width 1,2,4,8          */
  uint64_t section_off[VBQ_NSECTIONS];
  uint64_t section_len[VBQ_NSECTIONS];
  uint64_t total_bytes;  /* size of the blob                           */
  uint32_t flags;        /* call options (VBQ_Y_F16, ...); packers write 0 */
  uint32_t reserved1;
} vbq_desc;

/* Packing options; a zero field selects the library's choice. */
typedef struct vbq_pack_opts {
  int32_t tile_rows;     /* 0 or a power of two in [16, 256]           */
  int32_t chunk_groups;  /* 0 or 1..128 with tile_rows*chunk_groups <= 8192 */
  uint32_t flags;        /* reserved, 0                                */
  uint32_t n_threads;    /* host threads for packing; 0 = hardware     */
} vbq_pack_opts;

/* Human-readable name of a status code (static storage, never NULL). */
const char* vbq_status_string(vbq_status s);

/* Name of the last HIP runtime error that made an entry point of this thread
 * return VBQ_ERR_HIP ("hipSuccess" if none); static storage, never NULL. */
const char* vbq_last_hip_error(void);

/* Layout version this library reads and writes. */
uint32_t vbq_layout_version(void);

/* Bytes of the blob that vbq_pack / vbq_pack_codes would write for a matrix
 * with the given bit map.  bits: host uint8[N][K/64], each in {1,2,4,8}.
 * opts may be NULL.  Also fills *desc_out (may be NULL) with the layout. */
vbq_status vbq_pack_size(int64_t N, int64_t K, const uint8_t* bits,
                         const vbq_pack_opts* opts, size_t* bytes,
                         vbq_desc* desc_out);

/* Quantize and pack (paper section 3.1, Eq. (1) and the 1-bit rule).
 * W: host float32[N][K] row-major; bits: host uint8[N][K/64].
 * blob: host buffer of blob_bytes >= vbq_pack_size() bytes, 8-byte aligned.
 * On success fills *desc.  Errors: NULL, SHAPE, BITS, NONFINITE (NaN/Inf in
 * W), SCALE_RANGE (a scale that overflows fp16), BUFFER, UNSUPPORTED. */
vbq_status vbq_pack(int64_t N, int64_t K, const float* W, const uint8_t* bits,
                    const vbq_pack_opts* opts, void* blob, size_t blob_bytes,
                    vbq_desc* desc);

/* Pack already-quantized codes.  q: host int8[N][K] (levels, not offset
 * codes); scale_f16: host uint16[N][K/64] fp16 bit patterns; bits as above.
 * Errors additionally: CODE_RANGE (q outside the width's level set),
 * NONFINITE / SCALE_RANGE (scale is NaN/Inf or negative). */
vbq_status vbq_pack_codes(int64_t N, int64_t K, const int8_t* q,
                          const uint16_t* scale_f16, const uint8_t* bits,
                          const vbq_pack_opts* opts, void* blob,
                          size_t blob_bytes, vbq_desc* desc);

/* Check a descriptor against this library's layout (magic, version, shape,
 * section offsets inside total_bytes).  VBQ_OK or VBQ_ERR_DESC / NULL. */
vbq_status vbq_desc_check(const vbq_desc* d);

/* y[n] = sum_k w_hat[n][k] * x[k]   (fused dequantize + GEMV, paper section 6)
 * blob_dev: the packed blob in device memory (desc->total_bytes bytes,
 * 256-byte aligned); x_dev: device fp16[K], 16-byte aligned; y_dev: device
 * float32[N] (fp16[N] with VBQ_Y_F16).  Asynchronous on stream (a hipStream_t;
 * NULL = default stream).  The sum over each row is taken in a fixed order, so
 * results are bitwise reproducible for a given blob.  Errors: NULL, DESC,
 * BUFFER (misaligned), UNSUPPORTED (unknown flags, blob >= 4 GiB), HIP. */
vbq_status vbq_gemv(const vbq_desc* desc, const void* blob_dev,
                    const void* x_dev, void* y_dev, void* stream);

/* Row-bucketed output (paper section 6, "Fused kernels over packed weights":
 * the mixed-precision LM head is stored as a few frequency-grouped row
 * buckets; section 4, the recipe's frequency-tiered head).  As vbq_gemv, but
 * row n of this matrix is written to y_dev[row_index_dev[n]]: a bucket is
 * packed as its own matrix (one width, so no width map) and called with the
 * output rows of its members.  row_index_dev: device int32[N]; an index
 * outside [0, y_len) is not written (no error).  The indices of one call
 * should be distinct: rows sharing an index are all written to it, in no
 * defined order (the value is one of theirs).  The caller owns every buffer;
 * buckets of one output may run back to back on one stream.  Errors: NULL,
 * SHAPE (y_len < 0), BUFFER (misaligned pointers), DESC, HIP. */
vbq_status vbq_gemv_rows(const vbq_desc* desc, const void* blob_dev,
                         const void* x_dev, void* y_dev, int64_t y_len,
                         const int32_t* row_index_dev, void* stream);

/* ---------------------------------------------------------------------------
 * Row buckets (paper section 6, "Fused kernels over packed weights": the
 * mixed-precision LM head is stored as a few frequency-grouped row buckets;
 * section 4: the recipe's head gives each row one width by its token's
 * frequency rank).  A matrix whose rows each have ONE width is stored as one
 * packed matrix per width present (a bucket: one width, so no width map), and
 * each bucket writes its rows of y through vbq_gemv_rows.
 * ------------------------------------------------------------------------- */
#define VBQ_MAX_BUCKETS 4

typedef struct vbq_bucket {
  int32_t bits;          /* the bucket's width: 1, 2, 4 or 8                  */
  int32_t reserved;      /* 0                                                 */
  int64_t row_begin;     /* its rows' output indices are                     */
  int64_t n_rows;        /*   row_index[row_begin .. row_begin + n_rows)      */
  uint64_t blob_offset;  /* byte offset of its packed matrix in the blob     */
  vbq_desc desc;         /* its packed matrix: n_rows x K, all of width bits  */
} vbq_bucket;

/* Bytes of the blob vbq_pack_row_buckets writes, and the number of buckets
 * (widths present).  row_bits: host uint8[N], the width of every group of
 * row n, each in {1,2,4,8}.  opts as for vbq_pack (applied to every bucket;
 * NULL = the library's choice per bucket).  Errors: NULL, SHAPE, BITS,
 * UNSUPPORTED. */
vbq_status vbq_pack_row_buckets_size(int64_t N, int64_t K, const uint8_t* row_bits,
                                     const vbq_pack_opts* opts, size_t* bytes,
                                     int32_t* n_buckets);

/* Pack a matrix of one width per row as row buckets.  q: host int8[N][K]
 * levels; scale_f16: host uint16[N][K/64] fp16 scales; row_bits as above.
 * Bucket i (increasing width) holds the rows of that width in increasing row
 * order, packed exactly as vbq_pack_codes packs those rows alone (so its bytes
 * are that call's bytes), at blob + buckets[i].blob_offset (256-byte aligned).
 * row_index (host int32[N]) receives the rows of bucket 0, then bucket 1, ...
 * blob: host buffer of blob_bytes >= vbq_pack_row_buckets_size bytes, 8-byte
 * aligned.  Upload blob and row_index to the device as they are.  Errors:
 * NULL, SHAPE, BITS, CODE_RANGE, NONFINITE, SCALE_RANGE, BUFFER, UNSUPPORTED. */
vbq_status vbq_pack_row_buckets(int64_t N, int64_t K, const int8_t* q,
                                const uint16_t* scale_f16, const uint8_t* row_bits,
                                const vbq_pack_opts* opts, void* blob,
                                size_t blob_bytes,
                                vbq_bucket buckets[VBQ_MAX_BUCKETS],
                                int32_t* n_buckets, int32_t* row_index);

/* y = w_hat x for a bucketed matrix (paper section 6, the head stored as
 * frequency-grouped row buckets): bucket i reads blob_dev +
 * buckets[i].blob_offset and writes its rows to y[row_index_dev[row_begin +
 * n]], each row's value bit for bit that of vbq_gemv_rows on the bucket.
 * When two or more buckets each take the four-wave one-width kernel and all
 * carry the same flags (as vbq_pack_row_buckets' buckets of one call do),
 * every bucket runs in ONE launch (vbq_buckets_kernel<4>, the buckets side
 * by side); otherwise vbq_gemv_rows runs for each bucket in turn on the
 * stream.  The buckets' output rows must not overlap (with one launch, which
 * bucket's value lands in a shared row is unspecified).  The bucket
 * descriptors' flags apply.  blob_dev 256-byte aligned; row_index_dev device
 * int32[sum n_rows]; y_dev device float32[y_len] (fp16 with VBQ_Y_F16).
 * Errors: as vbq_gemv_rows, and SHAPE for n_buckets outside
 * [0, VBQ_MAX_BUCKETS]. */
vbq_status vbq_gemv_buckets(const vbq_bucket* buckets, int32_t n_buckets,
                            const void* blob_dev, const int32_t* row_index_dev,
                            const void* x_dev, void* y_dev, int64_t y_len,
                            void* stream);

/* Y[m][n] = sum_k w_hat[n][k] * X[m][k] for m < M, 0 <= M <= 16
 * (small-batch decode).  X_dev: device fp16 rows with stride ldx >= K
 * elements (ldx % 8 == 0); Y_dev: device float32 rows (fp16 with VBQ_Y_F16)
 * with stride ldy >= N elements.  M == 0 is a no-op.  Weights are streamed
 * once for all M rows. */
vbq_status vbq_gemm_small(const vbq_desc* desc, const void* blob_dev,
                          int64_t M, const void* X_dev, int64_t ldx,
                          void* Y_dev, int64_t ldy, void* stream);

/* ---------------------------------------------------------------------------
 * One launch per decode step (paper section 6, "The speedup grows with model
 * size": for small models the per-token overhead, not bandwidth, bounds
 * decode).  A step is a sequence of GEMVs in which GEMV i reads its x only
 * after every earlier GEMV of the step has written its y, as when x_i is
 * computed from y_(i-1).  vbq_step_run runs the whole sequence in one
 * cooperative launch: the weights of GEMV i are loaded while GEMV i-1 is
 * still running, and only x, the multiply and the store of y wait for it.
 * Each y is bitwise the y that vbq_gemv / vbq_gemv_rows give.
 * ------------------------------------------------------------------------- */
#define VBQ_STEP_MAX_GEMVS 65536

/* One GEMV of a step. */
typedef struct vbq_step_gemv {
  const vbq_desc* desc;  /* host descriptor of the packed matrix; its
                            VBQ_Y_F16 flag applies (VBQ_ONE_WAVE_PER_UNIT is
                            refused)                                         */
  const void* blob;      /* device blob, 256-byte aligned                    */
  const void* x;         /* device fp16[K], 16-byte aligned                  */
  void* y;               /* device float32 (fp16 with VBQ_Y_F16): y[N], or
                            y[y_len] written through rows                    */
  const int32_t* rows;   /* device int32[N] row map as in vbq_gemv_rows, or
                            NULL for y[n]                                    */
  int64_t y_len;         /* length of y when rows != NULL                    */
} vbq_step_gemv;

/* Bytes of the device plan of n GEMVs (1 <= n <= VBQ_STEP_MAX_GEMVS). */
vbq_status vbq_step_plan_bytes(int32_t n, size_t* bytes);

/* Bytes of the device workspace of vbq_step_run for n GEMVs: eight arrival
 * words per GEMV, each in its own 128-byte line (1 KiB per GEMV), then one
 * status word. */
vbq_status vbq_step_workspace_bytes(int32_t n, size_t* bytes);

/* Writes the plan of n GEMVs, run in array order, into plan_host (host
 * memory of plan_bytes >= vbq_step_plan_bytes bytes, 8-byte aligned).  The
 * caller copies it to device memory as it is; it stays valid while every
 * blob, x, y and rows buffer it names does.  Every matrix must have at most 8
 * units per row tile with at most 32 group columns each (the library's
 * default geometry for K <= 16384).  Errors: NULL, SHAPE, DESC, BUFFER
 * (misaligned buffers, plan too small), UNSUPPORTED (geometry outside that
 * range, VBQ_ONE_WAVE_PER_UNIT, unknown flags, blob >= 4 GiB). */
vbq_status vbq_step_plan(const vbq_step_gemv* gemvs, int32_t n, void* plan_host,
                         size_t plan_bytes);

/* Runs a plan of n GEMVs on stream: a small kernel that clears the workspace,
 * then one cooperative launch of one 16-wave workgroup per CU (the grid is
 * sized from the device's CU count and an occupancy query, and the launch
 * fails with VBQ_ERR_HIP rather than run a grid that does not fit).
 * plan_dev: the plan in device memory (8-byte aligned); workspace_dev: device
 * memory of workspace_bytes >= vbq_step_workspace_bytes (4-byte aligned),
 * caller-owned, not shared by runs that may overlap.  spin_limit bounds every
 * wait for an earlier GEMV (polls of about 0.1 us; 0 = 2^22): a workgroup that
 * reaches it stops waiting, skips its remaining work and sets the status word
 * (the workspace's last uint32) to 1, so the launch always ends; the status
 * word is 0 after a complete run.  Errors: NULL, SHAPE, BUFFER, HIP. */
vbq_status vbq_step_run(const void* plan_dev, int32_t n, void* workspace_dev,
                        size_t workspace_bytes, uint32_t spin_limit,
                        void* stream);

/* vbq_step_run without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops, harnesses that
 * forbid hipMalloc): the arrival words live in a scratch array the library
 * holds in device memory, 512 KiB per GPU it runs on, from the first call
 * on that GPU until the process ends.  No call allocates anything.
 *   n            1 .. 512 GEMVs (VBQ_ERR_SHAPE beyond; vbq_step_run has no
 *                such limit).
 *   status_dev   device uint32 (4-byte aligned) that receives the status word
 *                of vbq_step_run (0 complete, 1 a wait gave up), or NULL.
 * Every call on one GPU shares that GPU's scratch, which the call clears
 * first: calls that may overlap on one GPU (other streams, other threads)
 * race and must be serialized by the caller.  Errors: NULL, SHAPE, BUFFER,
 * UNSUPPORTED (device index >= 64), HIP. */
vbq_status vbq_step_run_noalloc(const void* plan_dev, int32_t n, uint32_t spin_limit,
                                uint32_t* status_dev, void* stream);

/* Name of the kernel that vbq_gemm_small with M activation rows (vbq_gemv and
 * vbq_gemv_rows for M = 1) launches on this matrix, named with its template
 * arguments as a profiler prints them without spaces, e.g.
 * "vbq_mv_pair_kernel<8,1>" (static storage; "none" for an invalid descriptor
 * or M outside [1, 16]).  The choice depends on the widths present, the grid
 * and the flags; a caller or a profile can group launches by it. */
const char* vbq_kernel_name(const vbq_desc* desc, int64_t M);

/* What vbq_gemv_buckets launches for these buckets: "vbq_buckets_kernel<4>"
 * (one launch for all of them), "per bucket" (vbq_gemv_rows for each; see
 * vbq_kernel_name) or "none" (n_buckets outside [1, VBQ_MAX_BUCKETS] or
 * NULL).  Static storage; only the descriptors are looked at. */
const char* vbq_gemv_buckets_kernel_name(const vbq_bucket* buckets, int32_t n_buckets);

/* W_dev[n][k] = w_hat[n][k] = s*q as float32 (exact), device float32[N][K].
 * For checking the packed stream against the quantizer bit for bit. */
vbq_status vbq_dequant(const vbq_desc* desc, const void* blob_dev,
                       float* W_dev, void* stream);

/* ---------------------------------------------------------------------------
 * Differentiable bit selection (training time; paper section 3.2 and
 * Algorithm 1).  These calls work on plain (unpacked) fp32 weights seen as a
 * flat array of n_groups groups of 64 contiguous weights: a row-major W[N][K]
 * with K % 64 == 0 is n_groups = N*K/64, and the concatenation of several such
 * matrices (a network's flat parameter buffer) can be passed as one array.
 * Candidate order everywhere is B = {1, 2, 4, 8} bits.
 * ------------------------------------------------------------------------- */

#define VBQ_QAT_MAX_GROUPS (((int64_t)1) << 40)
/* vbq_qat_forward flag: write w_soft as bf16 (each fp32 result rounded to
 * nearest even) instead of float. */
#define VBQ_QAT_WSOFT_BF16 1u

/* Bytes of device workspace vbq_qat_forward needs to compute bbar for
 * n_groups groups (8 bytes per block of its launch).  VBQ_ERR_NULL or
 * VBQ_ERR_SHAPE (n_groups < 0 or > VBQ_QAT_MAX_GROUPS). */
vbq_status vbq_qat_workspace_size(int64_t n_groups, size_t* bytes);

/* Forward pass of the selection path (paper section 3.2, Algorithm 1 lines of
 * the weight and logit steps that build w_hat).  For each group g:
 *   w_hat^(b)  = the per-group quantizer of section 3.1 at width b, exactly as
 *                vbq_pack applies it (Eq. (1) for b >= 2, sign/absmean for
 *                b = 1, fp16-rounded scale, round-half-to-even against the
 *                stored scale, sign(0) = +1), so a one-hot pi gives exactly the
 *                weights vbq_dequant returns after vbq_pack at that width;
 *   pi_g       = softmax((logits_g + noise_g) / tau) in fp32;
 *   w_soft_i   = sum_k pi_{g,k} * w_hat^(B_k)_i (fp32, FMA);
 *   hard_g     = B[argmax_k logits_{g,k}] (first of equal maxima; the noise
 *                does not enter), Algorithm 1's hardened width;
 *   bbar       = (1/n_groups) sum_g sum_k pi_{g,k} B_k (double), the expected
 *                bit cost of section 3.2.
 * Arguments (all device pointers, caller-owned; the call only enqueues work):
 *   W_dev        float[n_groups*64] weights, 16-byte aligned.  Each group's
 *                max|w| must be below 65520 (its 2-bit scale is an fp16 value);
 *                a group outside that range or with NaN/Inf gives non-finite
 *                outputs for that group (not checked).
 *   logits_dev   float[n_groups][4], 16-byte aligned.
 *   noise_dev    float[n_groups][4] Gumbel noise drawn by the caller, 16-byte
 *                aligned, or NULL for no noise (plain softmax).
 *   tau          temperature, finite and >= FLT_MIN (the smallest normal
 *                float); the softmax subtracts the group's largest l + e before
 *                dividing by tau, so any such tau gives finite pi.
 *   flags        0, or VBQ_QAT_WSOFT_BF16 for a bf16 w_soft; other bits give
 *                VBQ_ERR_UNSUPPORTED.
 *   w_soft_dev   float[n_groups*64] output (bf16[n_groups*64] with
 *                VBQ_QAT_WSOFT_BF16), 16-byte aligned; may not overlap the
 *                inputs.
 *   pi_dev       float[n_groups][4] output (16-byte aligned) or NULL.
 *   hard_bits_dev uint8[n_groups] output or NULL.
 *   bbar_dev     one double output (8-byte aligned) or NULL; needs a workspace
 *                of vbq_qat_workspace_size bytes (8-byte aligned), whose
 *                contents are scratch.  bbar is summed in a fixed order, so
 *                repeated calls give the same bits.
 * n_groups == 0 does nothing (any pointer may then be NULL; bbar is not
 * written).  Errors: VBQ_ERR_NULL (W, logits or w_soft NULL; workspace NULL
 * with bbar), VBQ_ERR_SHAPE (n_groups out of range),
 * VBQ_ERR_NONFINITE (tau NaN/Inf), VBQ_ERR_UNSUPPORTED (tau < FLT_MIN,
 * unknown flags), VBQ_ERR_BUFFER (misaligned pointer or workspace too small),
 * VBQ_ERR_HIP. */
vbq_status vbq_qat_forward(int64_t n_groups, const float* W_dev,
                           const float* logits_dev, const float* noise_dev,
                           float tau, uint32_t flags, void* w_soft_dev,
                           float* pi_dev, uint8_t* hard_bits_dev,
                           double* bbar_dev, void* workspace_dev,
                           size_t workspace_bytes, void* stream);

/* Gradient of the logit step (paper section 3.3, "Gradient isolation", and
 * Algorithm 1): the candidate reconstructions are held constant, so with
 * G = dL_CE/dw_soft the loss L = L_CE + lambda*bbar reaches the logits only
 * through pi:
 *   a_{g,k}     = sum_{i in g} G_i * w_hat^(B_k)_i + lambda * B_k / n_bbar
 *   dlogits_g,k = (pi_{g,k} / tau) * (a_{g,k} - sum_j pi_{g,j} * a_{g,j}).
 * The candidates are recomputed from W exactly as vbq_qat_forward forms them;
 * the sums over a group are fp32 FMAs.
 * Arguments (device pointers, caller-owned, 16-byte aligned; enqueued only):
 *   W_dev        float[n_groups*64] the weights of the forward pass.
 *   grad_dev     float[n_groups*64] dL_CE/dw_soft, same layout.
 *   pi_dev       float[n_groups][4] the forward's pi (same tau and noise).
 *   tau          the forward's temperature, finite and >= FLT_MIN.
 *   lambda       the bit penalty, finite.
 *   n_bbar       the n that divides bbar (>= 1): this array's n_groups for a
 *                per-matrix penalty, the network's total group count when the
 *                penalty is on the network's mean bits.
 *   dlogits_dev  float[n_groups][4] output.
 * n_groups == 0 does nothing (pointers may then be NULL).  Errors:
 * VBQ_ERR_SHAPE (n_groups out of range, n_bbar < 1), VBQ_ERR_NONFINITE (tau
 * or lambda NaN/Inf), VBQ_ERR_UNSUPPORTED (tau < FLT_MIN), VBQ_ERR_NULL,
 * VBQ_ERR_BUFFER (misaligned), VBQ_ERR_HIP. */
vbq_status vbq_qat_logit_grad(int64_t n_groups, const float* W_dev,
                              const float* grad_dev, const float* pi_dev,
                              float tau, float lambda, int64_t n_bbar,
                              float* dlogits_dev, void* stream);

/* ---------------------------------------------------------------------------
 * Measurement aid of the roofline harness (not part of the method).
 * ------------------------------------------------------------------------- */

/* Reads `bytes` bytes at src_dev (device, 16-byte aligned, bytes % 16 == 0)
 * with 16-byte non-temporal loads over `blocks` workgroups of 256 lanes
 * (0 = 8192), folding them with XOR into sink_dev (device uint32[4 * blocks],
 * contents meaningless), so the time of the launch is the device's plain
 * streaming-read rate.  Errors: NULL, BUFFER, UNSUPPORTED (blocks > 2^20), HIP. */
vbq_status vbq_read_ceiling(const void* src_dev, size_t bytes, uint32_t blocks,
                            uint32_t* sink_dev, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* VBQ_H */
