// The C-ABI entry points of include/nmm.h: argument checks, planning and launches.
// Every function validates everything before enqueueing anything and never throws.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>

#include "nmm_internal.h"

using namespace nmm;

namespace {

size_t rup256(size_t v) { return (v + 255) / 256 * 256; }
int64_t rup8(int64_t v) { return (v + 7) / 8 * 8; }

}  // namespace

// Compute units of the current device (256 on MI355X; also the answer when no device is visible),
// queried once per device and kept.
int nmm::device_cus() {
    constexpr int kDevices = 64;
    static std::atomic<int> cached[kDevices] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kDevices) return 256;
    int cus = cached[dev].load(std::memory_order_relaxed);
    if (cus > 0) return cus;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) cus = 256;
    cached[dev].store(cus, std::memory_order_relaxed);
    return cus;
}

namespace {

// The launches of one validated, planned GEMV on the workspace `ws`.
nmm_status gemv_launch(const GemvArgs& a, const GemvPlan& p, void* ws, void* stream) {
    unsigned* tickets = static_cast<unsigned*>(ws);
    float* part = ws ? reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + kTicketBytes) : nullptr;
    if (p.path == NMM_PATH_MFMA && a.K > 0) return launch_mfma(a, p, tickets, part, stream);
    return launch_gemv(a, p, tickets, part, stream);
}

nmm_status gemv_common(const GemvArgs& a, int path, void* ws, size_t ws_bytes, void* stream) {
    nmm_status st = validate_gemv(a, path);
    if (st != NMM_OK) return st;
    GemvPlan p;
    st = plan_gemv(a.batch, a.M, a.K, a.N, a.dt, path, &p);
    if (st != NMM_OK) return st;
    if (a.batch == 0 || a.M == 0 || a.N == 0) return NMM_OK;
    if (a.K > 0) {
        st = validate_workspace(ws, ws_bytes, p.ws_bytes);
        if (st != NMM_OK) return st;
    }
    return gemv_launch(a, p, ws, stream);
}

// ---------------------------------------------------------------------------------------------
// The allocation-free GEMV's scratch: one array per GPU in the library's device code, resolved to
// a device address once per device (hipGetSymbolAddress, with that device current) and kept.  Its
// first kTicketBytes are the split-K arrival counters: zeroed by a fill kernel on the first call
// on each device, and left at zero by every launch after it.
// ---------------------------------------------------------------------------------------------
constexpr size_t kScratchBytes = NMM_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];
constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kScratchDevices] = {};

nmm_status scratch_of_current_device(void** out, hipStream_t s) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kScratchDevices) return NMM_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return NMM_ERR_HIP;
        const nmm_status st = launch_zero_fill(ptr, kTicketBytes, s);
        if (st != NMM_OK) return st;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return NMM_OK;
}

// The five narrow MatMuls of one decode chain, with their fused bf16 hand-offs.  All steps
// share one workspace: each takes its own range of the counter block at the head (so every
// counter any call ever uses lies in that block) and its own partial-sum region after it.
struct Chain {
    GemvArgs step[5];
    GemvPlan plan[5];
    int64_t tick_off[5];   // first counter of each step
    size_t part_off[5];    // byte offset of each step's partial sums (from the workspace start)
    size_t ws_total;
};

bool chain_dims_ok(const nmm_mla_chain& c) {
    const int64_t d[] = {c.hidden, c.q_lora, c.kv_lora, c.rope, c.heads, c.nope, c.v_head};
    for (int64_t v : d)
        if (v <= 0 || v >= (int64_t(1) << 31)) return false;
    return c.nope + c.rope < (int64_t(1) << 31) / c.heads;
}

nmm_status build_chain(const nmm_mla_chain& c, Chain* out) {
    if (!chain_dims_ok(c)) return NMM_ERR_SHAPE;
    const int64_t n_down = c.q_lora + c.kv_lora + c.rope;
    const int64_t qk = c.nope + c.rope;
    Chain ch;
    GemvArgs* s = ch.step;
    // down = x . w_down ; c_q = bf16(down[:q_lora])
    s[0].K = c.hidden; s[0].N = n_down; s[0].x = c.x; s[0].ldx = c.hidden;
    s[0].w = c.w_down; s[0].ldw = n_down; s[0].y = c.down_f32; s[0].ldy = n_down;
    s[0].ybf = c.cq_bf16; s[0].ybf_group = n_down; s[0].ybf_keep = c.q_lora; s[0].ybf_ldm = c.q_lora;
    // q = c_q . w_uq ; q_nope = bf16(q[h, :nope])
    s[1].K = c.q_lora; s[1].N = c.heads * qk; s[1].x = c.cq_bf16; s[1].ldx = c.q_lora;
    s[1].w = c.w_uq; s[1].ldw = c.heads * qk; s[1].y = c.q_f32; s[1].ldy = c.heads * qk;
    s[1].ybf = c.qnope_bf16; s[1].ybf_group = qk; s[1].ybf_keep = c.nope; s[1].ybf_ldm = c.heads * c.nope;
    // lat[h] = q_nope[h] . w_uk[h] ; lat' = bf16(lat)
    s[2].batch = c.heads; s[2].K = c.nope; s[2].N = c.kv_lora;
    s[2].x = c.qnope_bf16; s[2].ldx = c.nope; s[2].sx = c.nope;
    s[2].w = c.w_uk; s[2].ldw = c.kv_lora; s[2].sw = c.nope * c.kv_lora;
    s[2].y = c.lat_f32; s[2].ldy = c.kv_lora; s[2].sy = c.kv_lora;
    s[2].ybf = c.lat_bf16; s[2].ybf_group = c.kv_lora; s[2].ybf_keep = c.kv_lora;
    s[2].ybf_ldm = c.kv_lora; s[2].ybf_sb = c.kv_lora;
    // o[h] = lat'[h] . w_uv[h] ; o' = bf16(o)
    s[3].batch = c.heads; s[3].K = c.kv_lora; s[3].N = c.v_head;
    s[3].x = c.lat_bf16; s[3].ldx = c.kv_lora; s[3].sx = c.kv_lora;
    s[3].w = c.w_uv; s[3].ldw = c.v_head; s[3].sw = c.kv_lora * c.v_head;
    s[3].y = c.o_f32; s[3].ldy = c.v_head; s[3].sy = c.v_head;
    s[3].ybf = c.o_bf16; s[3].ybf_group = c.v_head; s[3].ybf_keep = c.v_head;
    s[3].ybf_ldm = c.v_head; s[3].ybf_sb = c.v_head;
    // y = o' . w_o
    s[4].K = c.heads * c.v_head; s[4].N = c.hidden; s[4].x = c.o_bf16; s[4].ldx = c.heads * c.v_head;
    s[4].w = c.w_o; s[4].ldw = c.hidden; s[4].y = c.y; s[4].ldy = c.hidden;
    size_t off = kTicketBytes;
    int64_t ticks = 0;
    for (int i = 0; i < 5; ++i) {
        s[i].M = 1;
        s[i].dt = NMM_BF16;
        nmm_status st = plan_gemv(s[i].batch, 1, s[i].K, s[i].N, NMM_BF16, NMM_PATH_GEMV, &ch.plan[i]);
        if (st != NMM_OK) return st;
        ch.tick_off[i] = ticks;
        ch.part_off[i] = off;
        if (ch.plan[i].split()) {
            ticks += ch.plan[i].n_tickets;
            off += rup256(static_cast<size_t>(ch.plan[i].part_floats) * 4);
        }
    }
    if (ticks > kMaxTickets) return NMM_ERR_SHAPE;
    ch.ws_total = off;   // the counter block is always part of it
    *out = ch;
    return NMM_OK;
}

// MatMul 2 and its cache entry: the GEMV's arguments and plan, and the workspace they need (the
// counter block always, for the epilogue's panel counter).
struct KvUpdate {
    GemvArgs args;
    GemvPlan plan;
    size_t ws_bytes = 0;
};

// The cache entry's own arguments (shared by nmm_mla_kv_update and the chain).
nmm_status validate_kv_entry(int64_t kv_lora, int64_t rope, float eps, float theta, int64_t position,
                             int64_t ld_cache, int64_t cache_rows, int round) {
    constexpr int64_t kLim = int64_t(1) << 31;
    if (kv_lora <= 0 || rope < 0 || (rope & 1) || kv_lora + rope > kKvMaxWidth || rope > kKvMaxRope)
        return NMM_ERR_SHAPE;
    if (ld_cache < kv_lora + rope || cache_rows <= 0 || ld_cache >= kLim) return NMM_ERR_SHAPE;
    if (position < 0 || position >= cache_rows) return NMM_ERR_SHAPE;
    if (!std::isfinite(eps) || eps < 0.f || !std::isfinite(theta) || theta <= 0.f) return NMM_ERR_ARG;
    if (round != NMM_ROUND_EVEN && round != NMM_ROUND_AWAY) return NMM_ERR_ARG;
    return NMM_OK;
}

KvEpilogue kv_epilogue(const void* gamma, float eps, float theta, int64_t position, void* cache, int64_t ld_cache,
                       int64_t c_off, int64_t kv_lora, int64_t rope, int round, unsigned* done) {
    KvEpilogue e;
    e.gamma = gamma;
    e.row = static_cast<uint16_t*>(cache) + position * ld_cache;
    e.done = done;
    e.eps = eps;
    e.theta = theta;
    e.position = position;
    e.c_off = c_off;
    e.kv = static_cast<int>(kv_lora);
    e.rope = static_cast<int>(rope);
    e.away = round == NMM_ROUND_AWAY ? 1 : 0;
    return e;
}

nmm_status build_kv_update(const nmm_mla_kv& k, KvUpdate* out) {
    constexpr int64_t kLim = int64_t(1) << 31;
    if (k.hidden <= 0 || k.hidden >= kLim) return NMM_ERR_SHAPE;
    nmm_status vst = validate_kv_entry(k.kv_lora, k.rope, k.eps, k.rope_theta, k.position, k.ld_cache, k.cache_rows,
                                       k.round);
    if (vst != NMM_OK) return vst;
    const int64_t n = k.kv_lora + k.rope;
    if (k.ldw < n) return NMM_ERR_SHAPE;
    KvUpdate u;
    GemvArgs& a = u.args;
    a.M = 1; a.K = k.hidden; a.N = n; a.dt = NMM_BF16;
    a.x = k.h; a.ldx = rup8(k.hidden); a.w = k.w; a.ldw = k.ldw; a.y = k.mm; a.ldy = n;
    nmm_status st = plan_gemv(1, 1, a.K, a.N, NMM_BF16, NMM_PATH_GEMV, &u.plan);
    if (st != NMM_OK) return st;
    if (u.plan.n_tickets + 1 > kMaxTickets) return NMM_ERR_SHAPE;
    u.ws_bytes = std::max<size_t>(u.plan.ws_bytes, kTicketBytes);
    *out = u;
    return NMM_OK;
}

}  // namespace

extern "C" {

nmm_status nmm_gemv(int64_t M, int64_t K, int64_t N, nmm_dtype dt, const void* x, int64_t ldx,
                    const void* W, int64_t ldw, float* y, int64_t ldy, nmm_path path,
                    void* workspace, size_t workspace_bytes, void* stream) {
    GemvArgs a;
    a.M = M; a.K = K; a.N = N; a.dt = dt;
    a.x = x; a.ldx = ldx; a.w = W; a.ldw = ldw; a.y = y; a.ldy = ldy;
    return gemv_common(a, path, workspace, workspace_bytes, stream);
}

nmm_status nmm_gemv_noalloc(int64_t M, int64_t K, int64_t N, nmm_dtype dt, const void* x, int64_t ldx,
                            const void* W, int64_t ldw, float* y, int64_t ldy, nmm_path path, void* stream) {
    GemvArgs a;
    a.M = M; a.K = K; a.N = N; a.dt = dt;
    a.x = x; a.ldx = ldx; a.w = W; a.ldw = ldw; a.y = y; a.ldy = ldy;
    nmm_status st = validate_gemv(a, path);
    if (st != NMM_OK) return st;
    GemvPlan p;
    st = plan_gemv(1, M, K, N, dt, path, &p);
    if (st != NMM_OK) return st;
    if (M == 0 || N == 0) return NMM_OK;
    void* ws = nullptr;
    if (K > 0 && p.ws_bytes > 0) {
        if (p.ws_bytes > kScratchBytes) return NMM_ERR_WORKSPACE;
        st = scratch_of_current_device(&ws, static_cast<hipStream_t>(stream));
        if (st != NMM_OK) return st;
    }
    return gemv_launch(a, p, ws, stream);
}

nmm_status nmm_batched_gemv(int64_t batch, int64_t M, int64_t K, int64_t N, nmm_dtype dt,
                            const void* x, int64_t ldx, int64_t stride_x,
                            const void* W, int64_t ldw, int64_t stride_w,
                            float* y, int64_t ldy, int64_t stride_y, nmm_path path,
                            void* workspace, size_t workspace_bytes, void* stream) {
    GemvArgs a;
    a.batch = batch; a.M = M; a.K = K; a.N = N; a.dt = dt;
    a.x = x; a.ldx = ldx; a.sx = stride_x;
    a.w = W; a.ldw = ldw; a.sw = stride_w;
    a.y = y; a.ldy = ldy; a.sy = stride_y;
    return gemv_common(a, path, workspace, workspace_bytes, stream);
}

nmm_status nmm_gemv_bf16(int64_t M, int64_t K, int64_t N, nmm_dtype dt, const void* x, int64_t ldx,
                         const void* W, int64_t ldw, void* y_bf16, int64_t ldyb, nmm_round round,
                         float* y, int64_t ldy, nmm_path path, void* workspace, size_t workspace_bytes,
                         void* stream) {
    if (round != NMM_ROUND_EVEN && round != NMM_ROUND_AWAY) return NMM_ERR_ARG;
    GemvArgs a;
    a.M = M; a.K = K; a.N = N; a.dt = dt;
    a.x = x; a.ldx = ldx; a.w = W; a.ldw = ldw;
    a.y = y; a.ldy = y ? ldy : 0;
    if (M > 0 && N > 0 && !y_bf16) return NMM_ERR_NULL;
    if (ldyb < N) return NMM_ERR_SHAPE;
    // one group spanning every column: ybf[m * ldyb + n]
    a.ybf = y_bf16; a.ybf_group = std::max<int64_t>(N, 1); a.ybf_keep = a.ybf_group; a.ybf_ldm = ldyb;
    a.ybf_away = round == NMM_ROUND_AWAY ? 1 : 0;
    return gemv_common(a, path, workspace, workspace_bytes, stream);
}

nmm_status nmm_gemv_nt(int64_t M, int64_t K, int64_t N, nmm_dtype dt, const void* x, int64_t ldx,
                       const void* Wt, int64_t ldwt, float* y, int64_t ldy, void* workspace,
                       size_t workspace_bytes, void* stream) {
    GemvArgs a;
    a.M = M; a.K = K; a.N = N; a.dt = dt;
    a.x = x; a.ldx = ldx; a.w = Wt; a.ldw = ldwt; a.y = y; a.ldy = ldy;
    nmm_status st = validate_gemv_nt(a);
    if (st != NMM_OK) return st;
    NtPlan p;
    st = plan_gemv_nt(M, K, N, &p);
    if (st != NMM_OK) return st;
    if (M == 0 || N == 0) return NMM_OK;
    if (K > 0) {
        st = validate_workspace(workspace, workspace_bytes, p.ws_bytes);
        if (st != NMM_OK) return st;
    }
    unsigned* tickets = static_cast<unsigned*>(workspace);
    float* part = workspace ? reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + kTicketBytes) : nullptr;
    return launch_gemv_nt(a, p, p.ks > 1 ? tickets : nullptr, p.ks > 1 ? part : nullptr, stream);
}

size_t nmm_gemv_nt_workspace_size(int64_t M, int64_t K, int64_t N, nmm_dtype dt) {
    (void)dt;
    NtPlan p;
    return plan_gemv_nt(M, K, N, &p) == NMM_OK ? p.ws_bytes : 0;
}

nmm_status nmm_batched_gemv_bf16(int64_t batch, int64_t M, int64_t K, int64_t N, nmm_dtype dt,
                                 const void* x, int64_t ldx, int64_t stride_x,
                                 const void* W, int64_t ldw, int64_t stride_w,
                                 void* y_bf16, int64_t ldyb, int64_t stride_yb, nmm_round round,
                                 float* y, int64_t ldy, int64_t stride_y, nmm_path path,
                                 void* workspace, size_t workspace_bytes, void* stream) {
    if (round != NMM_ROUND_EVEN && round != NMM_ROUND_AWAY) return NMM_ERR_ARG;
    GemvArgs a;
    a.batch = batch; a.M = M; a.K = K; a.N = N; a.dt = dt;
    a.x = x; a.ldx = ldx; a.sx = stride_x;
    a.w = W; a.ldw = ldw; a.sw = stride_w;
    a.y = y; a.ldy = y ? ldy : 0; a.sy = y ? stride_y : 0;
    if (batch > 0 && M > 0 && N > 0 && !y_bf16) return NMM_ERR_NULL;
    if (ldyb < N || stride_yb < 0) return NMM_ERR_SHAPE;
    a.ybf = y_bf16; a.ybf_group = std::max<int64_t>(N, 1); a.ybf_keep = a.ybf_group; a.ybf_ldm = ldyb;
    a.ybf_sb = stride_yb;
    a.ybf_away = round == NMM_ROUND_AWAY ? 1 : 0;
    return gemv_common(a, path, workspace, workspace_bytes, stream);
}

nmm_status nmm_mla_query(int64_t heads, int64_t nope, int64_t rope, int64_t kv_lora, const float* q,
                         const void* q_bf16, const void* w_uk, int64_t position, float rope_theta,
                         float* qlat_f32, void* q_out, int64_t ldq, void* workspace, size_t workspace_bytes,
                         void* stream) {
    constexpr int64_t kLim = int64_t(1) << 31;
    if (heads < 0 || nope <= 0 || rope < 0 || (rope & 1) || rope > kKvMaxRope || kv_lora <= 0 || heads >= kLim ||
        kv_lora >= kLim || nope + rope >= kLim / std::max<int64_t>(heads, 1))
        return NMM_ERR_SHAPE;
    if (heads == 0) return NMM_OK;
    if (!q || !q_bf16 || !w_uk || !qlat_f32 || !q_out) return NMM_ERR_NULL;
    if (ldq < kv_lora + rope || ldq >= kLim || position < 0 || position >= kLim) return NMM_ERR_SHAPE;
    if (!std::isfinite(rope_theta) || rope_theta <= 0.f) return NMM_ERR_ARG;
    if ((reinterpret_cast<uintptr_t>(q) & 3u) || (reinterpret_cast<uintptr_t>(q_out) & 1u)) return NMM_ERR_ALIGN;
    // lat[h] = q_nope[h] . w_uk[h], q_nope = the first nope values of each head's bf16 query
    GemvArgs a;
    a.batch = heads; a.M = 1; a.K = nope; a.N = kv_lora; a.dt = NMM_BF16;
    a.x = q_bf16; a.ldx = nope; a.sx = nope + rope;
    a.w = w_uk; a.ldw = kv_lora; a.sw = nope * kv_lora;
    a.y = qlat_f32; a.ldy = kv_lora; a.sy = kv_lora;
    a.ybf = q_out; a.ybf_group = kv_lora; a.ybf_keep = kv_lora; a.ybf_ldm = ldq; a.ybf_sb = ldq;
    nmm_status st = validate_gemv(a, NMM_PATH_GEMV);
    if (st != NMM_OK) return st;
    GemvPlan p;
    st = plan_gemv(heads, 1, nope, kv_lora, NMM_BF16, NMM_PATH_GEMV, &p);
    if (st != NMM_OK) return st;
    st = validate_workspace(workspace, workspace_bytes, p.ws_bytes);
    if (st != NMM_OK) return st;
    unsigned* tickets = p.split() ? static_cast<unsigned*>(workspace) : nullptr;
    float* part = p.split() ? reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + kTicketBytes) : nullptr;
    return launch_gemv_qrope(a, p, tickets, part, q, q_out, ldq, static_cast<int>(heads), static_cast<int>(nope),
                             static_cast<int>(kv_lora), static_cast<int>(rope), position, rope_theta, stream);
}

}  // extern "C"

namespace {

// The three launches of nmm_mla_query_path with their plans.
struct QueryPath {
    GemvArgs down, uq, uk;
    GemvPlan p_down, p_uq, p_uk;
    size_t ws_bytes = 0;
};

nmm_status build_query_path(const nmm_mla_query_path& c, QueryPath* out) {
    constexpr int64_t kLim = int64_t(1) << 31;
    const int64_t d[] = {c.hidden, c.q_lora, c.kv_lora, c.heads, c.nope};
    for (int64_t v : d)
        if (v <= 0 || v >= kLim) return NMM_ERR_SHAPE;
    if (c.rope < 0 || (c.rope & 1) || c.rope > kKvMaxRope || c.nope + c.rope >= kLim / c.heads) return NMM_ERR_SHAPE;
    const int64_t n_down = c.q_lora + c.kv_lora + c.rope, qk = c.nope + c.rope;
    QueryPath q;
    q.down.K = c.hidden; q.down.N = n_down; q.down.x = c.x; q.down.ldx = c.hidden;
    q.down.w = c.w_down; q.down.ldw = n_down; q.down.y = c.down_f32; q.down.ldy = n_down;
    q.down.ybf = c.cq_bf16; q.down.ybf_group = n_down; q.down.ybf_keep = c.q_lora; q.down.ybf_ldm = c.q_lora;
    q.uq.K = c.q_lora; q.uq.N = c.heads * qk; q.uq.x = c.cq_bf16; q.uq.ldx = c.q_lora;
    q.uq.w = c.w_uq; q.uq.ldw = c.heads * qk; q.uq.y = c.q_f32; q.uq.ldy = c.heads * qk;
    q.uq.ybf = c.q_bf16; q.uq.ybf_group = c.heads * qk; q.uq.ybf_keep = c.heads * qk; q.uq.ybf_ldm = c.heads * qk;
    q.uk.batch = c.heads; q.uk.K = c.nope; q.uk.N = c.kv_lora; q.uk.x = c.q_bf16; q.uk.ldx = c.nope; q.uk.sx = qk;
    q.uk.w = c.w_uk; q.uk.ldw = c.kv_lora; q.uk.sw = c.nope * c.kv_lora;
    q.uk.y = c.qlat_f32; q.uk.ldy = c.kv_lora; q.uk.sy = c.kv_lora;
    q.uk.ybf = c.query; q.uk.ybf_group = c.kv_lora; q.uk.ybf_keep = c.kv_lora; q.uk.ybf_ldm = c.ldq; q.uk.ybf_sb = c.ldq;
    GemvArgs* a[] = {&q.down, &q.uq, &q.uk};
    GemvPlan* p[] = {&q.p_down, &q.p_uq, &q.p_uk};
    for (int i = 0; i < 3; ++i) {
        a[i]->M = 1;
        a[i]->dt = NMM_BF16;
        nmm_status st = plan_gemv(a[i]->batch, 1, a[i]->K, a[i]->N, NMM_BF16, NMM_PATH_GEMV, p[i]);
        if (st != NMM_OK) return st;
        q.ws_bytes = std::max(q.ws_bytes, p[i]->ws_bytes);
    }
    *out = q;
    return NMM_OK;
}

}  // namespace

namespace {

AttnArgs attn_args(const nmm_latent_attn& l) {
    AttnArgs a;
    a.heads = l.heads; a.seq = l.seq; a.d_qk = l.d_qk; a.d_v = l.d_v;
    a.q = l.q; a.ldq = l.ldq; a.kv = l.kv; a.ld_kv = l.ld_kv; a.scale = l.scale;
    a.out = l.out; a.ldo = l.ldo; a.outb = l.out_bf16; a.ldob = l.ldob; a.splits = l.splits;
    return a;
}

struct Span {
    uintptr_t lo = 0, hi = 0;   // [lo, hi) in bytes; empty when lo == hi
};
Span span_of(const void* p, int64_t bytes) {
    Span s;
    if (p && bytes > 0) {
        s.lo = reinterpret_cast<uintptr_t>(p);
        s.hi = s.lo + static_cast<uintptr_t>(bytes);
    }
    return s;
}
bool overlaps(const Span& a, const Span& b) { return a.lo < a.hi && b.lo < b.hi && a.lo < b.hi && b.lo < a.hi; }

// The attention of a decode step runs concurrently with the chain, so neither may touch what the
// other writes.  Called with validated shapes (the chain built, the attention planned).
nmm_status validate_attention_independent(const nmm_mla_chain& c, const AttnArgs& a) {
    if (a.heads == 0) return NMM_OK;
    const int64_t lim = int64_t(1) << 31;
    if (a.ldq < a.d_qk || a.ldq >= lim || a.ld_kv < std::max(a.d_qk, a.d_v) || a.ld_kv >= lim || a.ldo < a.d_v ||
        a.ldo >= lim || (a.outb && (a.ldob < a.d_v || a.ldob >= lim)))
        return NMM_ERR_SHAPE;
    const int64_t n_down = c.q_lora + c.kv_lora + c.rope, qk = c.nope + c.rope;
    const Span writes[] = {
        span_of(c.down_f32, n_down * 4), span_of(c.q_f32, c.heads * qk * 4), span_of(c.lat_f32, c.heads * c.kv_lora * 4),
        span_of(c.o_f32, c.heads * c.v_head * 4), span_of(c.y, c.hidden * 4), span_of(c.cq_bf16, c.q_lora * 2),
        span_of(c.qnope_bf16, c.heads * c.nope * 2), span_of(c.lat_bf16, c.heads * c.kv_lora * 2),
        span_of(c.o_bf16, c.heads * c.v_head * 2),
        span_of(c.kv_cache ? static_cast<const uint8_t*>(c.kv_cache) + c.position * c.ld_cache * 2 : nullptr,
                (c.kv_lora + c.rope) * 2)};
    const Span reads[] = {
        span_of(c.x, c.hidden * 2), span_of(c.w_down, c.hidden * n_down * 2), span_of(c.w_uq, c.q_lora * c.heads * qk * 2),
        span_of(c.w_uk, c.heads * c.nope * c.kv_lora * 2), span_of(c.w_uv, c.heads * c.kv_lora * c.v_head * 2),
        span_of(c.w_o, c.heads * c.v_head * c.hidden * 2),
        span_of(c.kv_cache ? c.kv_gamma : nullptr, c.kv_lora * 2)};
    const Span att_in[] = {span_of(a.q, ((a.heads - 1) * a.ldq + a.d_qk) * 2),
                           span_of(a.kv, ((a.seq - 1) * a.ld_kv + std::max(a.d_qk, a.d_v)) * 2)};
    const Span att_out[] = {span_of(a.out, ((a.heads - 1) * a.ldo + a.d_v) * 4),
                            span_of(a.outb, ((a.heads - 1) * a.ldob + a.d_v) * 2)};
    for (const Span& w : writes) {
        for (const Span& r : att_in)
            if (overlaps(w, r)) return NMM_ERR_ARG;
        for (const Span& o : att_out)
            if (overlaps(w, o)) return NMM_ERR_ARG;
    }
    for (const Span& r : reads)
        for (const Span& o : att_out)
            if (overlaps(r, o)) return NMM_ERR_ARG;
    return NMM_OK;
}

}  // namespace

extern "C" {

size_t nmm_mla_query_path_workspace_size(const nmm_mla_query_path* qp) {
    if (!qp) return 0;
    QueryPath q;
    return build_query_path(*qp, &q) == NMM_OK ? q.ws_bytes : 0;
}

nmm_status nmm_mla_query_path_run(const nmm_mla_query_path* qp, void* workspace, size_t workspace_bytes,
                                  void* stream) {
    if (!qp) return NMM_ERR_NULL;
    const nmm_mla_query_path& c = *qp;
    if (!c.x || !c.w_down || !c.w_uq || !c.w_uk || !c.kv_gamma || !c.kv_cache || !c.down_f32 || !c.cq_bf16 ||
        !c.q_f32 || !c.q_bf16 || !c.qlat_f32 || !c.query)
        return NMM_ERR_NULL;
    QueryPath q;
    nmm_status st = build_query_path(c, &q);
    if (st != NMM_OK) return st;
    for (const GemvArgs* a : {&q.down, &q.uq, &q.uk}) {
        st = validate_gemv(*a, NMM_PATH_GEMV);
        if (st != NMM_OK) return st;
    }
    st = validate_kv_entry(c.kv_lora, c.rope, c.kv_eps, c.rope_theta, c.position, c.ld_cache, c.cache_rows, c.round);
    if (st != NMM_OK) return st;
    if (c.ldq < c.kv_lora + c.rope || c.ldq >= (int64_t(1) << 31)) return NMM_ERR_SHAPE;
    if (reinterpret_cast<uintptr_t>(c.kv_gamma) & 1u || reinterpret_cast<uintptr_t>(c.kv_cache) & 1u ||
        reinterpret_cast<uintptr_t>(c.query) & 1u)
        return NMM_ERR_ALIGN;
    st = validate_workspace(workspace, workspace_bytes, q.ws_bytes);
    if (st != NMM_OK) return st;
    unsigned* tickets = static_cast<unsigned*>(workspace);
    float* part = workspace ? reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + kTicketBytes) : nullptr;
    auto tk = [&](const GemvPlan& p) { return p.split() ? tickets : nullptr; };
    auto pt = [&](const GemvPlan& p) { return p.split() ? part : nullptr; };
    st = launch_gemv(q.down, q.p_down, tk(q.p_down), pt(q.p_down), stream);
    if (st != NMM_OK) return st;
    const KvEpilogue e = kv_epilogue(c.kv_gamma, c.kv_eps, c.rope_theta, c.position, c.kv_cache, c.ld_cache, c.q_lora,
                                     c.kv_lora, c.rope, c.round, nullptr);
    st = launch_gemv_entry(q.uq, q.p_uq, tk(q.p_uq), pt(q.p_uq), e, c.down_f32 + c.q_lora, stream);
    if (st != NMM_OK) return st;
    return launch_gemv_qrope(q.uk, q.p_uk, tk(q.p_uk), pt(q.p_uk), c.q_f32, c.query, c.ldq, static_cast<int>(c.heads),
                             static_cast<int>(c.nope), static_cast<int>(c.kv_lora), static_cast<int>(c.rope),
                             c.position, c.rope_theta, stream);
}

size_t nmm_mla_query_workspace_size(int64_t heads, int64_t nope, int64_t kv_lora) {
    GemvPlan p;
    return plan_gemv(heads, 1, nope, kv_lora, NMM_BF16, NMM_PATH_GEMV, &p) == NMM_OK ? p.ws_bytes : 0;
}

size_t nmm_gemv_workspace_size(int64_t M, int64_t K, int64_t N, nmm_dtype dt, nmm_path path) {
    GemvPlan p;
    return plan_gemv(1, M, K, N, dt, path, &p) == NMM_OK ? p.ws_bytes : 0;
}

size_t nmm_batched_gemv_workspace_size(int64_t batch, int64_t M, int64_t K, int64_t N,
                                       nmm_dtype dt, nmm_path path) {
    GemvPlan p;
    return plan_gemv(batch, M, K, N, dt, path, &p) == NMM_OK ? p.ws_bytes : 0;
}

nmm_status nmm_gemv_plan(int64_t batch, int64_t M, int64_t K, int64_t N, nmm_dtype dt,
                         nmm_path path, nmm_plan_info* info) {
    if (!info) return NMM_ERR_NULL;
    GemvPlan p;
    nmm_status st = plan_gemv(batch, M, K, N, dt, path, &p);
    if (st != NMM_OK) return st;
    info->path = p.path;
    info->m_tile = p.mt;
    info->m_blocks = p.mblocks;
    info->panel_width = p.cw_full;
    info->n_full_panels = p.n_full;
    info->tail_chunks = p.tail_chunks;
    info->tail_width = p.tail_cw;
    info->split_k_full = p.ks_full;
    info->rows_full = p.rows_full;
    info->split_k_tail = p.ks_tail;
    info->rows_tail = p.rows_tail;
    info->items = p.items;
    info->threads = kThreads;
    info->unroll = p.unroll;
    info->grid = p.grid;
    info->workspace_bytes = static_cast<int64_t>(p.ws_bytes);
    return NMM_OK;
}

size_t nmm_mla_decode_chain_workspace_size(const nmm_mla_chain* chain) {
    if (!chain) return 0;
    Chain ch;
    return build_chain(*chain, &ch) == NMM_OK ? ch.ws_total : 0;
}

}  // extern "C"

namespace {

// The chain's launches.  With `att`, the attention's workgroups share W_UQ's launch and its merge
// shares the W_UK -> W_UV pair's (W_O's where the pair runs as two batched GEMVs); with the cache
// entry, which takes a spare workgroup of W_UQ's launch, the attention shares W_O's launch and
// its merge follows.  The attention's workspace follows the chain's at a 256-byte boundary.
nmm_status run_chain(const nmm_mla_chain* chain, const AttnArgs* att, void* workspace, size_t workspace_bytes,
                     void* stream) {
    if (!chain) return NMM_ERR_NULL;
    const nmm_mla_chain& c = *chain;
    if (!c.x || !c.w_down || !c.w_uq || !c.w_uk || !c.w_uv || !c.w_o || !c.down_f32 || !c.q_f32 ||
        !c.lat_f32 || !c.o_f32 || !c.y || !c.cq_bf16 || !c.qnope_bf16 || !c.lat_bf16 || !c.o_bf16)
        return NMM_ERR_NULL;
    Chain ch;
    nmm_status st = build_chain(c, &ch);
    if (st != NMM_OK) return st;
    for (int i = 0; i < 5; ++i) {
        st = validate_gemv(ch.step[i], NMM_PATH_GEMV);
        if (st != NMM_OK) return st;
    }
    size_t att_ws = 0;
    if (att) {
        st = attention_workspace_bytes(*att, &att_ws);
        if (st != NMM_OK) return st;
    }
    const size_t att_off = rup256(ch.ws_total);
    st = validate_workspace(workspace, workspace_bytes, att ? att_off + att_ws : ch.ws_total);
    if (st != NMM_OK) return st;
    if (c.kv_cache) {
        if (!c.kv_gamma) return NMM_ERR_NULL;
        st = validate_kv_entry(c.kv_lora, c.rope, c.kv_eps, c.rope_theta, c.position, c.ld_cache, c.cache_rows,
                               c.round);
        if (st != NMM_OK) return st;
        if (reinterpret_cast<uintptr_t>(c.kv_gamma) & 1u || reinterpret_cast<uintptr_t>(c.kv_cache) & 1u)
            return NMM_ERR_ALIGN;
    }
    if (att) {
        st = validate_attention_args(*att, att_ws ? static_cast<uint8_t*>(workspace) + att_off : nullptr, att_ws);
        if (st != NMM_OK) return st;
        st = validate_attention_independent(c, *att);
        if (st != NMM_OK) return st;
    }
    if (c.events) {
        if (c.n_events < 6) return NMM_ERR_ARG;
        for (int i = 0; i < 6; ++i)
            if (!c.events[i]) return NMM_ERR_NULL;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    void* const att_mem = att_ws ? static_cast<uint8_t*>(workspace) + att_off : nullptr;
    // W_UK and W_UV run as one launch, one workgroup per head, where the dimensions allow it;
    // events 2 and 3 are then recorded together before it
    const bool pair = head_pair_ok(c.heads, c.nope, c.kv_lora, c.v_head);
    for (int i = 0; i < 5; ++i) {
        if (c.events && hipEventRecord(static_cast<hipEvent_t>(c.events[i]), s) != hipSuccess)
            return NMM_ERR_HIP;
        if (pair && i == 2) continue;
        if (pair && i == 3) {
            // with attention beside W_UQ, its merge on the compute units the pair's workgroups leave
            // free
            st = att && !c.kv_cache
                     ? launch_head_pair_merge(c.heads, c.nope, c.qnope_bf16, c.w_uk, c.w_uv, c.lat_f32, c.lat_bf16,
                                              c.o_f32, c.o_bf16, *att, att_mem, att_ws, stream)
                     : launch_head_pair(c.heads, c.nope, c.qnope_bf16, c.w_uk, c.w_uv, c.lat_f32, c.lat_bf16, c.o_f32,
                                        c.o_bf16, stream);
            if (st != NMM_OK) return st;
            continue;
        }
        unsigned* tickets = nullptr;
        float* part = nullptr;
        if (ch.plan[i].split()) {
            tickets = static_cast<unsigned*>(workspace) + ch.tick_off[i];
            part = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + ch.part_off[i]);
        }
        if (i == 1 && c.kv_cache) {
            // the cache entry of the down-projection's kv_lora | rope columns, built by one extra
            // workgroup of the W_UQ launch (down is complete by then)
            const KvEpilogue e = kv_epilogue(c.kv_gamma, c.kv_eps, c.rope_theta, c.position, c.kv_cache, c.ld_cache,
                                             c.q_lora, c.kv_lora, c.rope, c.round, nullptr);
            st = launch_gemv_entry(ch.step[1], ch.plan[1], tickets, part, e, c.down_f32 + c.q_lora, stream);
        } else if (i == 1 && att) {
            // attention's workgroups on the compute units W_UQ leaves free; its merge rides in the
            // pair's launch, or W_O's without the pair
            st = launch_gemv_beside_attention(ch.step[1], ch.plan[1], tickets, part, *att, att_mem, att_ws, stream);
        } else if (i == 4 && att && c.kv_cache) {
            st = launch_gemv_attention(ch.step[4], ch.plan[4], tickets, part, *att, att_mem, att_ws, stream);
        } else if (i == 4 && att && !pair) {
            st = launch_gemv_merge(ch.step[4], ch.plan[4], tickets, part, *att, att_mem, att_ws, stream);
        } else {
            st = launch_gemv(ch.step[i], ch.plan[i], tickets, part, stream);
        }
        if (st != NMM_OK) return st;
    }
    if (c.events && hipEventRecord(static_cast<hipEvent_t>(c.events[5]), s) != hipSuccess)
        return NMM_ERR_HIP;
    return NMM_OK;
}

}  // namespace

extern "C" {

nmm_status nmm_mla_decode_chain(const nmm_mla_chain* chain, void* workspace, size_t workspace_bytes, void* stream) {
    return run_chain(chain, nullptr, workspace, workspace_bytes, stream);
}

size_t nmm_mla_decode_step_workspace_size(const nmm_mla_chain* chain, const nmm_latent_attn* attn) {
    if (!chain || !attn) return 0;
    Chain ch;
    if (build_chain(*chain, &ch) != NMM_OK) return 0;
    size_t att_ws = 0;
    if (attention_workspace_bytes(attn_args(*attn), &att_ws) != NMM_OK) return 0;
    return rup256(ch.ws_total) + att_ws;
}

nmm_status nmm_mla_decode_step(const nmm_mla_chain* chain, const nmm_latent_attn* attn, void* workspace,
                               size_t workspace_bytes, void* stream) {
    if (!chain || !attn) return NMM_ERR_NULL;
    const AttnArgs a = attn_args(*attn);
    return run_chain(chain, &a, workspace, workspace_bytes, stream);
}

size_t nmm_mla_kv_update_workspace_size(const nmm_mla_kv* kv) {
    if (!kv) return 0;
    KvUpdate u;
    return build_kv_update(*kv, &u) == NMM_OK ? u.ws_bytes : 0;
}

nmm_status nmm_mla_kv_update(const nmm_mla_kv* kv, void* workspace, size_t workspace_bytes, void* stream) {
    if (!kv) return NMM_ERR_NULL;
    const nmm_mla_kv& k = *kv;
    if (!k.h || !k.w || !k.gamma || !k.mm || !k.cache) return NMM_ERR_NULL;
    KvUpdate u;
    nmm_status st = build_kv_update(k, &u);
    if (st != NMM_OK) return st;
    st = validate_gemv(u.args, NMM_PATH_GEMV);
    if (st != NMM_OK) return st;
    if (reinterpret_cast<uintptr_t>(k.gamma) & 1u || reinterpret_cast<uintptr_t>(k.cache) & 1u) return NMM_ERR_ALIGN;
    st = validate_workspace(workspace, workspace_bytes, u.ws_bytes);
    if (st != NMM_OK) return st;
    unsigned* counters = static_cast<unsigned*>(workspace);
    float* part = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + kTicketBytes);
    const KvEpilogue e = kv_epilogue(k.gamma, k.eps, k.rope_theta, k.position, k.cache, k.ld_cache, 0, k.kv_lora,
                                     k.rope, k.round, counters + u.plan.n_tickets);
    return launch_gemv_kv(u.args, u.plan, u.plan.split() ? counters : nullptr, u.plan.split() ? part : nullptr, e,
                          stream);
}

nmm_status nmm_workspace_init(void* workspace, size_t workspace_bytes, void* stream) {
    if (workspace_bytes == 0) return NMM_OK;
    if (!workspace) return NMM_ERR_NULL;
    if (reinterpret_cast<uintptr_t>(workspace) & 255u) return NMM_ERR_WORKSPACE;
    return launch_zero_fill(workspace, workspace_bytes, stream);
}

const char* nmm_status_string(nmm_status s) {
    switch (s) {
        case NMM_OK: return "NMM_OK";
        case NMM_ERR_NULL: return "NMM_ERR_NULL: a required pointer is NULL";
        case NMM_ERR_SHAPE: return "NMM_ERR_SHAPE: invalid size, leading dimension or stride";
        case NMM_ERR_DTYPE: return "NMM_ERR_DTYPE: unknown dtype";
        case NMM_ERR_ALIGN: return "NMM_ERR_ALIGN: pointer or leading dimension misaligned";
        case NMM_ERR_WORKSPACE: return "NMM_ERR_WORKSPACE: workspace missing, misaligned or too small";
        case NMM_ERR_HIP: return "NMM_ERR_HIP: HIP runtime error";
        case NMM_ERR_PATH: return "NMM_ERR_PATH: path unknown or unavailable for these sizes";
        case NMM_ERR_ARG: return "NMM_ERR_ARG: invalid argument";
    }
    return "unknown nmm_status";
}

const char* nmm_version(void) { return "0.1.0"; }

}  // extern "C"
