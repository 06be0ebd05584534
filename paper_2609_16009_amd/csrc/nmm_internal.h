// Internal declarations shared by the host planner, the C-ABI entry points and the kernels.
// Nothing here is part of the public ABI (include/nmm.h is).
#pragma once

#include <cstddef>
#include <cstdint>

#include "nmm.h"

namespace nmm {

// ---------------------------------------------------------------------------------------------
// Streaming GEMV geometry.
//
// W is read in 16-byte chunks (8 consecutive 16-bit columns of one row).  A "panel" is a column
// range of W: a full panel is cw_full chunks wide (64, 32, 16 or 8 chunks = 512..64 columns), and
// a wave folds 64 / cw_full rows into one step so that every lane issues one 16-byte load per
// step (1 KB per wave).  The ragged last panel has tail_chunks < cw_full chunks and folds
// 64 / tail_width rows (tail_width = a power of two >= tail_chunks).  Each workgroup owns one
// K-slice of one panel (a work "item").  Narrow panels give parallelism without deep K-splits,
// which keeps the partial-sum traffic and the final gather short.
// ---------------------------------------------------------------------------------------------
constexpr int kWaves = 4;                  // waves per GEMV workgroup
constexpr int kThreads = 64 * kWaves;      // threads per GEMV workgroup
constexpr int kPanelChunks = 64;           // chunks per full panel
constexpr int kPanelCols = 8 * kPanelChunks;
constexpr int kMaxMTile = 16;              // rows of x per GEMV launch
constexpr int kXStageBytes = 32 * 1024;    // LDS for the staged x slice of one item
constexpr int kRedBytes = 32 * 1024;       // LDS for the cross-wave reduction
// Every split-K workspace starts with a fixed block of arrival counters, and the partial sums
// always follow it.  So no call's partial sums can land on another call's counters, and one
// zeroed workspace serves any sequence of calls with different shapes.
constexpr int64_t kMaxTickets = 16384;
constexpr int64_t kTicketBytes = kMaxTickets * 4;

// Matrix-core path (mfma_gemv.hip): 128-column panels, W staged 64 rows at a time.
constexpr int kMfmaPanelCols = 128;
constexpr int kMfmaStageRows = 64;
constexpr int kMfmaTargetGrid = 256;      // the matrix-core plan splits K until about this many workgroups
constexpr int kMfmaMinMDefault = 3;        // AUTO uses the matrix cores from this many rows on

struct GemvPlan {
    int path = NMM_PATH_GEMV;
    int mt = 1;            // M tile (1, 2, 4, 8, 16)
    int mblocks = 1;       // ceil(M / mt)
    int unroll = 8;        // row steps in flight per wave
    int cw_full = kPanelChunks;  // chunks (= lanes per row) of a full panel: 64, 32, 16 or 8
    int n_full = 0;        // full panels
    int tail_chunks = 0;   // chunks in the last (ragged) panel, 0 if none
    int tail_cw = 0;       // lanes per row in the last panel (power of two >= tail_chunks)
    int ks_full = 0, rows_full = 0;
    int ks_tail = 0, rows_tail = 0;
    int ks_max = 1;        // max(ks_full, ks_tail)
    int items = 0;         // workgroups per (batch entry, row block)
    int64_t grid = 0;      // workgroups per launch
    int64_t n_tickets = 0; // arrival counters (one per panel per batch entry per row block)
    int64_t part_floats = 0;
    size_t ws_bytes = 0;   // kTicketBytes of counters + partial sums (0 when not split)
    bool split() const { return ks_max > 1; }
};

// Validated arguments of one (batched) GEMV launch.  Element strides.
struct GemvArgs {
    int64_t batch = 1, M = 0, K = 0, N = 0;
    int dt = NMM_BF16;
    const void* x = nullptr; int64_t ldx = 0, sx = 0;
    const void* w = nullptr; int64_t ldw = 0, sw = 0;
    float* y = nullptr; int64_t ldy = 0, sy = 0;
    // Optional fused bf16 copy of y: output column n goes to
    //   ybf[b*ybf_sb + m*ybf_ldm + (n / ybf_group) * ybf_keep + (n % ybf_group)]
    // when (n % ybf_group) < ybf_keep.
    void* ybf = nullptr; int64_t ybf_group = 0, ybf_keep = 0, ybf_ldm = 0, ybf_sb = 0;
    int ybf_away = 0;   // rounding of ybf: 0 nearest-even, 1 nearest with ties away from zero
};

// The cache entry behind MatMul 2 (gemv.hip): y[c_off .. c_off + kv + rope) of an M = 1 bf16 GEMV
// becomes row = bf16([RMSNorm(c) * gamma | RoPE(k, position)]).  `done` is a counter in the
// workspace's counter block, zero before and after the launch.
struct KvEpilogue {
    const void* gamma = nullptr;
    void* row = nullptr;
    unsigned* done = nullptr;
    float eps = 0.f, theta = 0.f;
    int64_t position = 0, c_off = 0;
    int kv = 0, rope = 0, away = 0;
};
constexpr int kKvMaxWidth = 4096;   // kv + rope values the epilogue stages in LDS
constexpr int kKvMaxRope = 512;     // RoPE width: one pair per thread of a 256-thread workgroup

// The transposed-weight GEMV (Wt row-major [N, K]): 4 r rows per workgroup, r per wave; K split
// into slices of slice_k (a multiple of 512) only where x's slice exceeds the LDS staging buffer.
struct NtPlan {
    int mt = 1, mblocks = 1;
    int r = 1, row_blocks = 1;
    int rgroup = 1;        // rows a wave walks together (1, 2, 4 or 8; r is a multiple of it)
    int depth = 8;         // loads in flight per lane: rgroup x steps (8, or 16 for 1-row tiles)
    int slice_k = 512, ks = 1;
    int64_t grid = 0;
    int64_t n_tickets = 0;
    size_t ws_bytes = 0;
};
nmm_status validate_gemv_nt(const GemvArgs& a);
nmm_status plan_gemv_nt(int64_t M, int64_t K, int64_t N, NtPlan* p);

// Pure host functions (no HIP calls): argument checks and the partition.
nmm_status validate_gemv(const GemvArgs& a, int path);
// unroll > 0 requests that many row-steps in flight (2, 4, 8, or 16 for tiles of <= 2 rows);
// 0 takes the default.
nmm_status plan_gemv(int64_t batch, int64_t M, int64_t K, int64_t N, int dt, int path, GemvPlan* p,
                     int unroll = 0);
nmm_status validate_workspace(const void* ws, size_t bytes, size_t need);

// Launchers (defined next to their kernels).  They assume validated arguments.
// `tickets` points into a workspace's counter block and `part` past it (both unused when the
// plan does not split K).
nmm_status launch_gemv(const GemvArgs& a, const GemvPlan& p, unsigned* tickets, float* part, void* stream);
nmm_status launch_zero_fill(void* ptr, size_t bytes, void* stream);
nmm_status launch_gemv_nt(const GemvArgs& a, const NtPlan& p, unsigned* tickets, float* part, void* stream);
// The GEMV of a validated M = 1 bf16 plan (path GEMV) followed in the same launch by the cache
// entry of `e` (K > 0).
nmm_status launch_gemv_kv(const GemvArgs& a, const GemvPlan& p, unsigned* tickets, float* part,
                          const KvEpilogue& e, void* stream);
// The GEMV of a validated M = 1 bf16 plan with one extra workgroup that builds the cache entry
// of `e` from src[0 .. kv + rope), a product an earlier launch on the stream completed.
nmm_status launch_gemv_entry(const GemvArgs& a, const GemvPlan& p, unsigned* tickets, float* part,
                             const KvEpilogue& e, const float* src, void* stream);
// A validated M = 1 bf16 batched GEMV plan with one extra workgroup that writes
// bf16(RoPE(q[h, nope : nope + rope], position)) to q_out[h * ldq + kv ..] for every head.
nmm_status launch_gemv_qrope(const GemvArgs& a, const GemvPlan& p, unsigned* tickets, float* part, const float* q,
                             void* q_out, int64_t ldq, int heads, int nope, int kv, int rope, int64_t position,
                             float theta, void* stream);
size_t gemv_kv_lds_bytes(const GemvPlan& p, int kv, int rope);

nmm_status launch_mfma(const GemvArgs& a, const GemvPlan& p, unsigned* tickets, float* part, void* stream);
size_t mfma_lds_bytes(const GemvPlan& p);
int device_cus();   // compute units of the current device

// The decode chain's W_UK -> W_UV pair in one launch, one workgroup per head (bf16, M = 1):
// usable for kv_lora 512, v_head 128 and nope a multiple of 4 * kPairUnroll up to 512.
constexpr int kPairUnroll = 16;
bool head_pair_ok(int64_t heads, int64_t nope, int64_t kv_lora, int64_t v_head);
nmm_status launch_head_pair(int64_t heads, int64_t nope, const void* q_nope, const void* w_uk, const void* w_uv,
                            float* lat, void* lat_bf16, float* o, void* o_bf16, void* stream);

// One latent-attention call (the arguments of nmm_latent_attention_ex).
struct AttnArgs {
    int64_t heads = 0, seq = 0, d_qk = 0, d_v = 0;
    const void* q = nullptr; int64_t ldq = 0;
    const void* kv = nullptr; int64_t ld_kv = 0;
    float scale = 1.f;
    float* out = nullptr; int64_t ldo = 0;
    void* outb = nullptr; int64_t ldob = 0;
    int64_t splits = 0;
};
// Workspace bytes of a valid call (0 when it needs none); NMM_ERR_* when the call is invalid.
nmm_status attention_workspace_bytes(const AttnArgs& a, size_t* bytes);
// Every check of the attention call, without launching.
nmm_status validate_attention_args(const AttnArgs& a, void* workspace, size_t workspace_bytes);
// The GEMV `g` (plain launch) and the attention `a` in one launch where both fit it (bf16, M = 1,
// the 576 / 512 attention shape, the GEMV's LDS within one attention chunk buffer): attention's
// workgroups first, then the GEMV's; then attention's merge launch.  Other shapes take the two launches in
// order.  The two must not touch each other's buffers.
nmm_status launch_gemv_attention(const GemvArgs& g, const GemvPlan& gp, unsigned* tickets, float* part,
                                 const AttnArgs& a, void* attn_ws, size_t attn_ws_bytes, void* stream);
// The same shared launch without the merge (the attention's span partials stay in its workspace),
// and a later GEMV launch that carries the merge: one extra workgroup per merge block in the
// GEMV's launch where the GEMV allows it, else the merge launch after the GEMV.  Between the two,
// nothing may write the attention's workspace or read its outputs.
nmm_status launch_gemv_beside_attention(const GemvArgs& g, const GemvPlan& gp, unsigned* tickets, float* part,
                                        const AttnArgs& a, void* attn_ws, size_t attn_ws_bytes, void* stream);
nmm_status launch_gemv_merge(const GemvArgs& g, const GemvPlan& gp, unsigned* tickets, float* part,
                             const AttnArgs& a, void* attn_ws, size_t attn_ws_bytes, void* stream);
// launch_head_pair carrying the merge of an attention launched earlier (as launch_gemv_merge):
// extra workgroups after the pair's run the merge blocks.
nmm_status launch_head_pair_merge(int64_t heads, int64_t nope, const void* q_nope, const void* w_uk, const void* w_uv,
                                  float* lat, void* lat_bf16, float* o, void* o_bf16, const AttnArgs& a,
                                  void* attn_ws, size_t attn_ws_bytes, void* stream);

}  // namespace nmm
