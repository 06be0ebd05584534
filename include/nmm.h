/*
 * nmm.h -- narrow MatMul on AMD MI355X (gfx950): the C ABI.
 *
 * The library computes narrow matrix multiplications y = x . W in which x has only a few rows
 * (any M on either path; AUTO streams W on the vector units for one row and uses the matrix
 * cores from three rows on, and from two where that needs no K-split), at the shapes of DeepSeek-V3
 * Multi-head Latent Attention single-token decode.  The operation is the paper's problem
 * statement C = A x B with A in R^{M x K}, B in R^{K x N}, narrow when min(M, N) = 1
 * (Section II-E "Problem Statement"; Section III-A, Condition 2 "Narrow Dimension"), widened to
 * small M as in the future-work Conditions 4-5 (Section V), and its specialisation C = T x W for
 * the MLA down-projection (Section IV-B, eq. 4).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - x and W hold 16-bit floats (fp16 or bf16, one type per call), row-major:
 *        x[m * ldx + k]  (m < M, k < K),     W[k * ldw + n]  (k < K, n < N).
 *    y is fp32, row-major, y[m * ldy + n], and is OVERWRITTEN (never accumulated into).
 *    Products are formed exactly in fp32 (16-bit inputs widen exactly) and summed in fp32.
 *  - All pointers except `stream` are device pointers on the current HIP device.  `stream` is a
 *    hipStream_t passed as void*; NULL means the null stream.  Calls are asynchronous: they
 *    enqueue kernels and return; results are valid once the stream's work completes.
 *  - The caller owns every buffer.  The library never allocates or frees memory in a compute
 *    call.  Buffers must stay alive until the enqueued work completes.
 *  - Alignment: x and W must be 16-byte aligned, and ldx and ldw must be multiples of 8
 *    elements (16 bytes).  A ragged N therefore needs a padded ldw >= roundup(N, 8); the kernels
 *    read the padding columns of each row (up to roundup(N, 8)) but never use them.  W's extent
 *    is (K-1)*ldw + roundup(N, 8) elements per matrix and x's is (M-1)*ldx + roundup(K, 8): reads
 *    are whole 16-byte chunks.  y needs 4-byte alignment only.
 *  - Workspace: split-K partial sums and arrival counters.  Query its size with the matching
 *    *_workspace_size() call; pass at least that many bytes, 256-byte aligned.  A workspace must
 *    be ZEROED once when it is allocated (nmm_workspace_init does that on a stream).  Its first
 *    64 KiB hold the arrival counters of every call and the partial sums always follow them;
 *    every call leaves the counters at zero again when it completes, so one workspace serves
 *    any sequence of calls of any shapes.  It serves one call at a time: calls that may overlap
 *    (different streams) need different workspaces.
 *  - Results are deterministic: the same inputs give bit-identical outputs on every run.
 *  - Errors: every call validates all arguments before enqueueing anything.  On an error it
 *    returns a non-zero nmm_status, enqueues nothing and leaves the outputs untouched.  No
 *    exception crosses the ABI and nothing aborts.  NMM_ERR_HIP reports that the HIP runtime
 *    returned an error after the call's launches (hipGetLastError): a failed launch, or an error
 *    an earlier runtime call on this thread left unread, which the call reads and so clears.
 *    A device-side fault surfaces at the caller's next synchronisation.
 *  - Empty problems: M == 0 or N == 0 is a no-op returning NMM_OK; K == 0 writes zeros (the
 *    empty sum).
 *  - Limits: every size and leading dimension must be < 2^31, each W matrix's extent must be
 *    < 2^31 bytes, and so must the x rows of one 32-row block, (min(M, 32) - 1) * ldx +
 *    roundup(K, 8) elements (buffer-resource offsets are 32-bit); otherwise NMM_ERR_SHAPE.
 */
#ifndef NMM_H
#define NMM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    NMM_OK = 0,
    NMM_ERR_NULL = 1,       /* a required pointer is NULL */
    NMM_ERR_SHAPE = 2,      /* negative size, ld smaller than the row, or a size over the limits */
    NMM_ERR_DTYPE = 3,      /* unknown nmm_dtype */
    NMM_ERR_ALIGN = 4,      /* a pointer or leading dimension breaks the alignment rules */
    NMM_ERR_WORKSPACE = 5,  /* workspace NULL, misaligned or smaller than the size query */
    NMM_ERR_HIP = 6,        /* the HIP runtime reported an error (no device, launch failure) */
    NMM_ERR_PATH = 7,       /* unknown nmm_path, or a path that cannot run these sizes */
    NMM_ERR_ARG = 8         /* any other invalid argument (e.g. non-finite attention scale) */
} nmm_status;

typedef enum { NMM_F16 = 1, NMM_BF16 = 2 } nmm_dtype;

/* Which kernel family computes the product.  AUTO picks from measured crossovers: the
 * streaming GEMV for M = 1, the MFMA (matrix-core) path for M >= 3, and at M = 2 the MFMA path
 * where its plan has a single K-slice (e.g. W_UQ [1536, 24576]), the GEMV otherwise (single
 * matrices; batched calls always stream).  GEMV and MFMA force a family.  NMM_PATH_MFMA with
 * batch > 1 is NMM_ERR_PATH.  The choice depends on the shape only. */
typedef enum { NMM_PATH_AUTO = 0, NMM_PATH_GEMV = 1, NMM_PATH_MFMA = 2 } nmm_path;

/*
 * nmm_gemv -- y[M,N] = x[M,K] . W[K,N].
 *
 * The paper's narrow MatMul (Section II-E; Condition 2) and its three-stage vector algorithm
 * (Algorithm 1, Section III-B: per-executor block loads, multiply + reduce to partial sums in a
 * temporary buffer, wait for all executors, gather).  Here the executors are workgroups: each
 * streams one K-slice of one column panel of W from HBM exactly once, keeps fp32 partial sums
 * per column, and the last workgroup to finish a panel gathers the K-slices in a fixed order
 * and writes y.
 *
 *   M, K, N     sizes (>= 0).  The GEMV path takes any M (in blocks of 16 rows); the MFMA path
 *               takes any M (in blocks of 32) for single matrices.
 *   dt          NMM_F16 or NMM_BF16, the type of both x and W.
 *   x, ldx      device pointer and leading dimension (elements, >= K, multiple of 8).
 *   W, ldw      device pointer and leading dimension (elements, >= N, multiple of 8).
 *   y, ldy      fp32 output and its leading dimension (elements, >= N).
 *   path        kernel family (see nmm_path).
 *   workspace   device scratch of >= nmm_gemv_workspace_size(...) bytes (may be NULL when that
 *               size is 0), zeroed once at allocation.
 *   stream      hipStream_t or NULL.
 */
nmm_status nmm_gemv(int64_t M, int64_t K, int64_t N, nmm_dtype dt,
                    const void* x, int64_t ldx, const void* W, int64_t ldw,
                    float* y, int64_t ldy, nmm_path path,
                    void* workspace, size_t workspace_bytes, void* stream);

/*
 * nmm_gemv_noalloc -- nmm_gemv without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses that forbid it).  It
 * allocates nothing on any call: the split-K counters and partial sums live in a scratch array of
 * NMM_NOALLOC_SCRATCH_BYTES in the library's device code, one per GPU, held until the process
 * ends.  Its counters are zeroed by a fill kernel on `stream` at the first call on each device and
 * every launch leaves them at zero.  Same arguments, rules and results as nmm_gemv (the same plan
 * and kernels, so the same bits); NMM_ERR_WORKSPACE when the plan needs more scratch than the
 * array holds (nmm_gemv_workspace_size(M, K, N, dt, path) > NMM_NOALLOC_SCRATCH_BYTES, e.g. the
 * streaming path at 16 rows of a [16384, 7168] weight), before anything is enqueued.  All calls
 * on one GPU share its array: calls that may overlap on one GPU (other streams, other host
 * threads) race and must not be made.
 */
#define NMM_NOALLOC_SCRATCH_BYTES ((size_t)8 << 20)
nmm_status nmm_gemv_noalloc(int64_t M, int64_t K, int64_t N, nmm_dtype dt,
                            const void* x, int64_t ldx, const void* W, int64_t ldw,
                            float* y, int64_t ldy, nmm_path path, void* stream);

/*
 * nmm_batched_gemv -- for b < batch: y_b = x_b . W_b with
 *   x_b = x + b*stride_x,  W_b = W + b*stride_w,  y_b = y + b*stride_y   (strides in elements).
 * The per-head absorbed MLA matmuls (q_nope . W_UK and latent . W_UV, one W per head).  Same
 * rules as nmm_gemv; stride_x and stride_w must be multiples of 8.  Strides may be smaller
 * than a matrix (e.g. a strided slice of a wider tensor); the caller guarantees y_b regions do
 * not overlap.
 */
nmm_status nmm_batched_gemv(int64_t batch, int64_t M, int64_t K, int64_t N, nmm_dtype dt,
                            const void* x, int64_t ldx, int64_t stride_x,
                            const void* W, int64_t ldw, int64_t stride_w,
                            float* y, int64_t ldy, int64_t stride_y, nmm_path path,
                            void* workspace, size_t workspace_bytes, void* stream);

/* Rounding of bf16 outputs: nearest with ties to even, or nearest with ties away from zero.
 * The paper's output cast (Algorithm 2, Section IV-E) is named CAST_ROUND without a definition,
 * so both nearest modes are offered; ties to even is the default reading. */
typedef enum { NMM_ROUND_EVEN = 0, NMM_ROUND_AWAY = 1 } nmm_round;

/*
 * nmm_gemv_bf16 -- y_bf16[M,N] = bf16(x[M,K] . W[K,N]): nmm_gemv's fp32 sums, rounded once to
 * bf16 in the same launch (Algorithm 2's output cast, Section IV-E; Alg. 2 returns C in bf16).
 *
 *   y_bf16, ldyb  bf16 output, y_bf16[m * ldyb + n]; 2-byte aligned, ldyb >= N (elements).
 *   round         NMM_ROUND_EVEN or NMM_ROUND_AWAY (anything else: NMM_ERR_ARG).
 *   y, ldy        optional fp32 copy of the same sums (NULL for none; ldy is then ignored).
 *
 * Everything else is as for nmm_gemv, including the workspace (nmm_gemv_workspace_size of the
 * same shape) and both kernel families.  K == 0 writes +0.
 */
nmm_status nmm_gemv_bf16(int64_t M, int64_t K, int64_t N, nmm_dtype dt,
                         const void* x, int64_t ldx, const void* W, int64_t ldw,
                         void* y_bf16, int64_t ldyb, nmm_round round,
                         float* y, int64_t ldy, nmm_path path,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * nmm_batched_gemv_bf16 -- nmm_batched_gemv with the sums also rounded once to bf16:
 * y_bf16[b*stride_yb + m*ldyb + n] (ldyb >= N, 2-byte aligned), ties per `round`; y (fp32, with
 * ldy and stride_y) may be NULL.  The per-head W_UV of the absorbed MLA step, whose bf16 output
 * feeds W_O.  Workspace as nmm_batched_gemv_workspace_size.
 */
nmm_status nmm_batched_gemv_bf16(int64_t batch, int64_t M, int64_t K, int64_t N, nmm_dtype dt,
                                 const void* x, int64_t ldx, int64_t stride_x,
                                 const void* W, int64_t ldw, int64_t stride_w,
                                 void* y_bf16, int64_t ldyb, int64_t stride_yb, nmm_round round,
                                 float* y, int64_t ldy, int64_t stride_y, nmm_path path,
                                 void* workspace, size_t workspace_bytes, void* stream);

/*
 * nmm_mla_query -- the absorbed MLA query of one token (the q path's end, Section IV-A's Cube
 * work that does not depend on MatMul 2), in one launch.  For each head h:
 *   q_out[h*ldq + c]           = bf16(sum_d q_nope[h,d] * W_UK[h][d, c])      c < kv_lora
 *   q_out[h*ldq + kv_lora + i] = bf16(RoPE(q[h, nope : nope+rope], position)[i])   i < rope
 * where q (fp32) and q_bf16 are W_UQ's output [heads, nope + rope] and its bf16 rounding, and
 * q_nope = q_bf16[h, :nope].  qlat_f32[h*kv_lora + c] receives the fp32 products.  RoPE as in
 * nmm_mla_kv_update (adjacent pairs, angle position * rope_theta^(-2i/rope)).  q_out is the
 * query nmm_latent_attention takes (d_qk = kv_lora + rope).
 *   heads >= 0; nope > 0 with nope and nope + rope multiples of 8; rope even, <= 512;
 *   ldq >= kv_lora + rope; q 4-byte, q_bf16 and w_uk 16-byte, q_out 2-byte aligned.
 * Workspace: nmm_mla_query_workspace_size(heads, nope, kv_lora).
 */
nmm_status nmm_mla_query(int64_t heads, int64_t nope, int64_t rope, int64_t kv_lora, const float* q,
                         const void* q_bf16, const void* w_uk, int64_t position, float rope_theta,
                         float* qlat_f32, void* q_out, int64_t ldq, void* workspace,
                         size_t workspace_bytes, void* stream);

/*
 * nmm_mla_query_path -- everything of one MLA decode step that precedes attention, in three
 * launches on one stream, MI355X's form of the paper's overlap (Section IV-A): MatMul 2 shares
 * its input with the query's down-projection, so both run as one GEMV, and the vector work
 * behind MatMul 2 runs on a spare workgroup of the next launch instead of on separate units.
 *   down    = x . w_down              [hidden, q_lora + kv_lora + rope]; c_q = bf16(down[:q_lora])
 *   q       = c_q . w_uq              q_f32 and its bf16 rounding q_bf16 [heads*(nope+rope)]
 *   kv_cache[position] = bf16([RMSNorm(down[q_lora : +kv_lora]) | RoPE(down[q_lora+kv_lora :])])
 *                                     (one extra workgroup of the W_UQ launch)
 *   query   = nmm_mla_query(q, q_bf16, w_uk)   [heads, ldq] bf16, qlat_f32 [heads*kv_lora]
 * Fields as in nmm_mla_decode_chain, nmm_mla_kv_update and nmm_mla_query (same limits; every
 * buffer required).  Workspace: nmm_mla_query_path_workspace_size.
 */
typedef struct {
    int64_t hidden, q_lora, kv_lora, rope, heads, nope;
    const void *x, *w_down, *w_uq, *w_uk, *kv_gamma;
    float kv_eps, rope_theta;
    int64_t position;
    void* kv_cache;
    int64_t ld_cache, cache_rows;
    nmm_round round;
    float* down_f32;   /* [q_lora + kv_lora + rope] */
    void* cq_bf16;     /* [q_lora] */
    float* q_f32;      /* [heads*(nope+rope)] */
    void* q_bf16;      /* [heads*(nope+rope)] */
    float* qlat_f32;   /* [heads*kv_lora] */
    void* query;       /* [heads, ldq] bf16 */
    int64_t ldq;
} nmm_mla_query_path;

nmm_status nmm_mla_query_path_run(const nmm_mla_query_path* qp, void* workspace, size_t workspace_bytes,
                                  void* stream);

/*
 * nmm_gemv_nt -- y[M,N] = x[M,K] . Wt[N,K]^T: the same product with W given transposed, row-major
 * [N, K] (Wt[n * ldwt + k]), the layout of a torch Linear weight and the one a dense
 * y = x . Wt^T GEMM reads, so one weight copy serves both (the paper keeps the matrix-unit
 * path's weight layout in global memory, Section IV-C; its Algorithm 1 multiplies rows by
 * columns).  Each output is the dot product of two contiguous rows: a wave streams 512 k of a
 * few Wt rows per step (two for one x row, four for more) with several steps in flight, and
 * folds its lanes at the end of the rows.  K is split (partials in
 * the workspace, combined in slice order in the same launch) only beyond 16384 / mt values,
 * mt = min(M, 4) rounded up to 1, 2 or 4; M above 4 runs in blocks of 4 rows, each reading Wt
 * again.
 *
 *   x, ldx      as for nmm_gemv (16-byte aligned, ldx >= K, multiple of 8).
 *   Wt, ldwt    16-byte aligned, ldwt >= K and a multiple of 8; (N-1)*ldwt + roundup(K, 8)
 *               elements < 2^31 bytes.  Values past K in a row's last 16 bytes are read, masked.
 *   y, ldy      fp32 output, ldy >= N.
 *   workspace   >= nmm_gemv_nt_workspace_size(M, K, N, dt) bytes (0 when K is not split).
 * Errors and empty problems as for nmm_gemv.
 */
nmm_status nmm_gemv_nt(int64_t M, int64_t K, int64_t N, nmm_dtype dt,
                       const void* x, int64_t ldx, const void* Wt, int64_t ldwt,
                       float* y, int64_t ldy, void* workspace, size_t workspace_bytes, void* stream);

/*
 * nmm_mla_kv_update -- DeepSeek-V3 MLA's MatMul 2 for one token and the vector work the paper
 * places behind it (Section IV-A: eq. 1 c^KV = W^DKV h, eq. 2 k^R = RoPE(W^KR h), eq. 3 the two
 * as one product; then RMSNorm, RoPE and caching), in one launch:
 *
 *   mm       = h . W                  W = (W^DKV | W^KR)^T  [hidden, kv_lora + rope]  (eq. 4)
 *   c'       = c / sqrt(mean(c^2) + eps) * gamma,      c = mm[:kv_lora]              (RMSNorm)
 *   k'[2i]   = k[2i] cos(a_i) - k[2i+1] sin(a_i)       k = mm[kv_lora:]              (RoPE on
 *   k'[2i+1] = k[2i] sin(a_i) + k[2i+1] cos(a_i)       a_i = position * theta^(-2i/rope)  adjacent
 *   cache[position, 0 : kv_lora + rope] = bf16([c' | k'])                              pairs)
 *
 * RMSNorm follows Zhang and Sennrich's definition and RoPE RoFormer's (the paper names both
 * without formulas).  W streams as in nmm_gemv (fp32 sums, K-slices added in slice order); the
 * last workgroup to finish gathers the slices of every column and builds the entry in fp32 (RoPE
 * angles formed and reduced modulo 2*pi in fp64) and rounds each value once to bf16 per `round`.  The layout of the entry is the latent cache that
 * nmm_latent_attention reads (V = its first kv_lora columns).
 *
 * Fields (NMM_ERR_SHAPE, _ALIGN, _ARG or _NULL before any launch):
 *   hidden, kv_lora, rope  > 0, > 0, even in [0, 512]; kv_lora + rope <= 4096.
 *   h          [hidden] bf16 token, 16-byte aligned; the kernel reads whole 16-byte chunks up to
 *              roundup(hidden, 8) elements (values past hidden are not used).
 *   w, ldw     W above, bf16, 16-byte aligned, ldw >= kv_lora + rope and a multiple of 8.
 *   gamma      [kv_lora] bf16 RMSNorm weight (2-byte aligned).
 *   eps        finite, >= 0.          rope_theta   finite, > 0.
 *   position   the token's position (its RoPE angle and its cache row), 0 <= position < cache_rows.
 *   mm         [kv_lora + rope] fp32: MatMul 2's product, an output.
 *   cache      bf16 latent cache [cache_rows, ld_cache], 2-byte aligned, ld_cache >= kv_lora +
 *              rope; only row `position`, columns [0, kv_lora + rope), is written.
 *   round      NMM_ROUND_EVEN or NMM_ROUND_AWAY.
 * The workspace (nmm_mla_kv_update_workspace_size) holds the split-K partials and the arrival
 * counters, the epilogue's among them; zeroed once at allocation, it is left zeroed.
 */
typedef struct {
    int64_t hidden, kv_lora, rope;   /* DeepSeek-V3: 7168, 512, 64 */
    const void* h;
    const void* w;
    int64_t ldw;
    const void* gamma;
    float eps, rope_theta;
    int64_t position;
    float* mm;
    void* cache;
    int64_t ld_cache, cache_rows;
    nmm_round round;
} nmm_mla_kv;

nmm_status nmm_mla_kv_update(const nmm_mla_kv* kv, void* workspace, size_t workspace_bytes,
                             void* stream);

/*
 * One DeepSeek-V3 MLA single-token decode chain of narrow MatMuls, all bf16 row-major [K,N]:
 *
 *   down   = x . w_down              x [1,hidden], w_down [hidden, q_lora+kv_lora+rope]
 *   c_q    = bf16(down[:q_lora])
 *   q      = c_q . w_uq              w_uq [q_lora, heads*(nope+rope)]
 *   q_nope = bf16(q[h, :nope])       per head h (the first nope of each head's nope+rope)
 *   lat[h] = q_nope[h] . w_uk[h]     w_uk [heads, nope, kv_lora]
 *   lat'   = bf16(lat)
 *   o[h]   = lat'[h] . w_uv[h]       w_uv [heads, kv_lora, v_head]
 *   o'     = bf16(o)                 flattened to [1, heads*v_head]
 *   y      = o' . w_o                w_o [heads*v_head, hidden]
 *
 * The first step is the paper's MatMul 2 (eq. 3, Section IV-A; eq. 4, Section IV-B), widened
 * from the kv_lora | rope columns to q_lora | kv_lora | rope.  Rounding to bf16 (ties to even) between steps
 * follows Algorithm 2's output cast (Section IV-E); it is fused into the producing kernel's
 * gather, which writes both the fp32 result and the bf16 operand of the next step.
 *
 * Every buffer is caller-owned device memory.  The fp32 and bf16 intermediates are outputs so
 * that each step can be checked on its own.  `events`, if not NULL, points to n_events >= 6
 * hipEvent_t handles; event i is recorded on `stream` before step i (i < 5) and event 5 after
 * the last step -- optional instrumentation for per-step timing.  When kv_lora = 512,
 * v_head = 128 and nope is a multiple of 64 up to 512, the two per-head steps run as one
 * launch (one workgroup per head) and events 2 and 3 are both recorded before it; other
 * dimensions take two batched launches.  Either way every output is the fp32 sum of the same
 * products; only the order of the additions differs between the two forms.
 *
 * Optionally (kv_cache not NULL) the chain also builds the latent cache entry from the
 * down-projection's kv_lora | rope columns, computed as nmm_mla_kv_update computes it:
 *   kv_cache[position, :kv_lora + rope] = bf16([RMSNorm(down[q_lora : q_lora + kv_lora]) |
 *                                               RoPE(down[q_lora + kv_lora :], position)])
 * with kv_gamma, kv_eps, rope_theta and round as there (same limits, NMM_ERR_* before any
 * launch).  One extra workgroup of the W_UQ launch builds it (down is complete by then), so no
 * step of the chain waits for it; the chain then always runs as separate launches.
 */
typedef struct {
    int64_t hidden, q_lora, kv_lora, rope, heads, nope, v_head;   /* 7168,1536,512,64,128,128,128 */
    const void *x, *w_down, *w_uq, *w_uk, *w_uv, *w_o;           /* bf16 inputs (see above)     */
    float *down_f32;   /* [q_lora+kv_lora+rope] */
    float *q_f32;      /* [heads*(nope+rope)]   */
    float *lat_f32;    /* [heads*kv_lora]       */
    float *o_f32;      /* [heads*v_head]        */
    float *y;          /* [hidden]  final output */
    void *cq_bf16;     /* [q_lora]             bf16 */
    void *qnope_bf16;  /* [heads*nope]         bf16 */
    void *lat_bf16;    /* [heads*kv_lora]      bf16 */
    void *o_bf16;      /* [heads*v_head]       bf16 */
    void *const *events;
    int n_events;
    /* optional cache entry behind the down-projection (see above) */
    const void* kv_gamma;          /* [kv_lora] bf16 RMSNorm weight */
    float kv_eps, rope_theta;
    int64_t position;
    void* kv_cache;                /* bf16 [cache_rows, ld_cache], or NULL for no entry */
    int64_t ld_cache, cache_rows;
    nmm_round round;
} nmm_mla_chain;

nmm_status nmm_mla_decode_chain(const nmm_mla_chain* chain, void* workspace,
                                size_t workspace_bytes, void* stream);

/*
 * nmm_latent_attention -- single-token latent attention, the decode step's independent dense
 * work (the paper overlaps the vector unit's narrow MatMul with matrix-unit work that does not
 * depend on it: Condition 1 "Data Independence", Section III-A; Section IV-A).  For each head h:
 *     s_j      = scale * sum_{d < d_qk} q[h*ldq + d] * kv[j*ld_kv + d]        (j < seq)
 *     p_j      = softmax_j(s)
 *     out[h,n] = sum_j p_j * kv[j*ld_kv + n]                                  (n < d_v)
 * i.e. V is the first d_v columns of the latent cache.  q and kv are bf16; out is fp32 with
 * leading dimension ldo.  Scores and softmax are fp32; p is rounded to bf16 for the matrix-core
 * product with V, accumulated in fp32.  Constraints (NMM_ERR_SHAPE / _ALIGN / _ARG before any
 * launch): heads >= 0, seq >= 1, d_qk a multiple of 32 in [32, 1024], d_v a multiple of 16 in
 * [16, 512], ld_kv >= max(d_qk, d_v), ldq >= d_qk, ldo >= d_v; ldq and ld_kv multiples of 8 and
 * ldo a multiple of 4; q and kv 16-byte aligned, out 16-byte aligned; finite scale.  Results are
 * deterministic for a given shape (fixed span partition and summation order); the workspace
 * (nmm_latent_attention_workspace_size) holds per-span partial results.
 */
nmm_status nmm_latent_attention(int64_t heads, int64_t seq, int64_t d_qk, int64_t d_v,
                                const void* q, int64_t ldq, const void* kv, int64_t ld_kv,
                                float scale, float* out, int64_t ldo,
                                void* workspace, size_t workspace_bytes, void* stream);

/* nmm_latent_attention with the partition chosen by the caller: `splits` position spans, each
 * taken by every block of heads (0: the default, min(ceil(seq / 128), max(64 / ceil(heads / 32),
 * ceil(seq / 512), min(floor(ceil(seq / 64) / 4), F))) spans with F = 256 / ceil(heads / 16), a multiple of 8
 * from 8 on, at most 64: at 4096 positions 16 for 128 heads and 32 for 16 to 64, at 8192
 * positions 32 for 128 heads, at 16384 32 for 128 heads and 64 for 16 to 64, from 32768 on 64;
 * the span is rounded up to whole 64-position chunks, so fewer spans may result), and an optional
 * bf16 copy of the output (out_bf16 may be NULL).  The launch takes blocks of 16 heads, and at
 * d_qk 576 / d_v 512 four or two workgroups per block and span (each a share of d_v's columns)
 * while that fits one workgroup per compute unit: 256 workgroups for 128 heads at the default.
 * Where even one workgroup per 16-head block and span would exceed 256 (128 heads from 32768
 * positions on), it takes blocks of 32 heads.  On MI355X at
 * 128 heads x 4096 positions attention alone is fastest with the default 16 spans, and so is the
 * decode step (nmm_mla_decode_step), whose attention workgroups take blocks of 32 heads beside an
 * HBM-bound stream.  The results depend on the spans only, not on the workgroups.  Workspace:
 * nmm_latent_attention_ex_workspace_size with the same splits. */
nmm_status nmm_latent_attention_ex(int64_t heads, int64_t seq, int64_t d_qk, int64_t d_v,
                                   const void* q, int64_t ldq, const void* kv, int64_t ld_kv,
                                   float scale, float* out, int64_t ldo, void* out_bf16, int64_t ldob,
                                   int64_t splits, void* workspace, size_t workspace_bytes, void* stream);

/* nmm_latent_attention, also writing out_bf16[h*ldob + n] = bf16(out[h*ldo + n]) (ties to even;
 * ldob >= d_v, 2-byte aligned): the operand of the per-head W_UV that follows attention. */
nmm_status nmm_latent_attention_bf16(int64_t heads, int64_t seq, int64_t d_qk, int64_t d_v,
                                     const void* q, int64_t ldq, const void* kv, int64_t ld_kv,
                                     float scale, float* out, int64_t ldo, void* out_bf16, int64_t ldob,
                                     void* workspace, size_t workspace_bytes, void* stream);

/*
 * nmm_mla_decode_step -- one decode step: the chain of nmm_mla_decode_chain and an independent
 * latent attention (the arguments of nmm_latent_attention_ex) on one stream, with the attention
 * run beside the chain's MatMuls instead of after them.  The paper's decode overlaps the narrow
 * MatMuls with matrix-unit work that does not depend on them (Condition 1 "Data Independence",
 * Section III-A; Section IV-A).  Here the overlap is fixed by the launches: the attention's
 * workgroups (blocks of 32 heads over the splits position spans) share W_UQ's grid, the GEMV's streaming
 * the weight while attention's use the compute units it leaves free, and the merge of the spans
 * rides on extra workgroups of the W_UK -> W_UV pair's launch (of W_O's where the pair runs as two
 * batched GEMVs).  With the cache entry (kv_cache), whose workgroup takes W_UQ's launch, the
 * attention shares W_O's launch instead and its merge follows in a launch of its own.  This needs
 * d_qk = 576, d_v = 512 and the chain's MatMuls in their single-row bf16 form; other shapes run the
 * attention in its own launches (same results).
 *
 * Results: every chain output as nmm_mla_decode_chain writes it, and out / out_bf16 as
 * nmm_latent_attention_ex writes them for the same splits (the same kernels' arithmetic).  The
 * attention must be independent of the chain: its q, kv, out and out_bf16 may not overlap any
 * buffer the chain writes (the cache row included), and out / out_bf16 no buffer the chain reads
 * (NMM_ERR_ARG).  Same limits as the two calls; `events` as in nmm_mla_decode_chain (each is
 * recorded before the launch that carries its MatMul, event 5 after the last launch).  Workspace:
 * nmm_mla_decode_step_workspace_size.
 */
typedef struct {
    int64_t heads, seq, d_qk, d_v;   /* DeepSeek-V3: 128 heads, 576, 512 */
    const void* q;                   /* bf16 [heads, ldq] */
    int64_t ldq;
    const void* kv;                  /* bf16 [seq, ld_kv] latent cache */
    int64_t ld_kv;
    float scale;
    float* out;                      /* fp32 [heads, ldo] */
    int64_t ldo;
    void* out_bf16;                  /* optional bf16 copy [heads, ldob], or NULL */
    int64_t ldob;
    int64_t splits;                  /* position spans (0: the default) */
} nmm_latent_attn;

nmm_status nmm_mla_decode_step(const nmm_mla_chain* chain, const nmm_latent_attn* attn, void* workspace,
                               size_t workspace_bytes, void* stream);

/* Workspace sizes in bytes (0 when none is needed; never fails: invalid sizes give 0). */
size_t nmm_gemv_workspace_size(int64_t M, int64_t K, int64_t N, nmm_dtype dt, nmm_path path);
size_t nmm_batched_gemv_workspace_size(int64_t batch, int64_t M, int64_t K, int64_t N,
                                       nmm_dtype dt, nmm_path path);
size_t nmm_mla_decode_chain_workspace_size(const nmm_mla_chain* chain);
size_t nmm_latent_attention_workspace_size(int64_t heads, int64_t seq, int64_t d_qk, int64_t d_v);
size_t nmm_mla_kv_update_workspace_size(const nmm_mla_kv* kv);
size_t nmm_gemv_nt_workspace_size(int64_t M, int64_t K, int64_t N, nmm_dtype dt);
size_t nmm_mla_query_workspace_size(int64_t heads, int64_t nope, int64_t kv_lora);
size_t nmm_mla_query_path_workspace_size(const nmm_mla_query_path* qp);
size_t nmm_latent_attention_ex_workspace_size(int64_t heads, int64_t seq, int64_t d_qk, int64_t d_v, int64_t splits);
size_t nmm_mla_decode_step_workspace_size(const nmm_mla_chain* chain, const nmm_latent_attn* attn);

/* Zero a workspace on `stream` with a fill kernel (no memset node, so it is safe to capture). */
nmm_status nmm_workspace_init(void* workspace, size_t workspace_bytes, void* stream);

/*
 * The host-side partition the library would launch for these sizes (a pure function: no GPU
 * access).  Algorithm 2's init stage (Section IV-E) sizes its executor pool from the core
 * count; here the plan sizes a grid of workgroups for 256 compute units.
 */
typedef struct {
    int32_t path;            /* NMM_PATH_GEMV or NMM_PATH_MFMA */
    int32_t m_tile;          /* rows of x per launch (GEMV: 1,2,4,8,16; MFMA: 16 or 32) */
    int32_t m_blocks;        /* launches' worth of row blocks (ceil(M / m_tile)) */
    int32_t panel_width;     /* 8-column chunks per full panel (64, 32, 16 or 8) */
    int32_t n_full_panels;   /* full panels */
    int32_t tail_chunks;     /* 8-column chunks in the ragged last panel (0: none) */
    int32_t tail_width;      /* lanes per row for the last panel (a power of two >= tail_chunks) */
    int32_t split_k_full;    /* K-slices per full panel */
    int32_t rows_full;       /* rows of W per K-slice of a full panel */
    int32_t split_k_tail;    /* K-slices of the last panel */
    int32_t rows_tail;       /* rows per K-slice of the last panel */
    int32_t items;           /* workgroups per matrix (per batch entry, per row block) */
    int32_t threads;         /* threads per workgroup */
    int32_t unroll;          /* row steps each wave keeps in flight */
    int64_t grid;            /* total workgroups of one launch */
    int64_t workspace_bytes;
} nmm_plan_info;

nmm_status nmm_gemv_plan(int64_t batch, int64_t M, int64_t K, int64_t N, nmm_dtype dt,
                         nmm_path path, nmm_plan_info* info);

/*
 * nmm_read_probe -- measurement support, not part of the product path: reads `bytes` (a multiple
 * of 16) of device memory at `buf` once with the GEMV's load instruction (16-byte non-temporal
 * buffer loads, `unroll` = 1, 2, 4 or 8 in flight per lane) on `grid` workgroups of 256 threads,
 * and writes one checksum word per workgroup to out[grid].  Timing it gives the practical HBM
 * read bandwidth that roofline fractions are compared against.
 */
nmm_status nmm_read_probe(const void* buf, size_t bytes, uint32_t* out, int64_t grid, int unroll,
                          void* stream);

/* Human-readable name of a status code (static storage). */
const char* nmm_status_string(nmm_status s);

/* Library version, e.g. "0.1.0" (static storage). */
const char* nmm_version(void);

#ifdef __cplusplus
}
#endif
#endif /* NMM_H */
