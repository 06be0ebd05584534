// Single-token latent attention on the matrix cores (gfx950), the decode step's independent
// dense work.  The paper's point is that narrow MatMuls moved off the matrix unit let
// independent matrix-unit work start earlier (Condition 1 "Data Independence", Section III-A;
// Section IV-A); this kernel is that independent work here, run on its own or with its workgroups
// beside the last narrow MatMul's in one launch (the decode step).
//
//   s_j = scale * q_h . kv_j[:d_qk],  p = softmax(s),  out_h = sum_j p_j kv_j[:d_v]
//
// Design (flash-decoding, one wave per 16 heads):
//  * A workgroup owns 64 heads and a span of positions; each of its 4 waves owns 16 of the heads
//    end to end.  The wave keeps its Q rows in registers as MFMA fragments.
//  * The span is walked in chunks of CH positions.  A chunk's cache rows (the first
//    max(d_qk, d_v) columns) are staged in LDS by buffer loads that write LDS directly, into one
//    of two buffers while the four waves compute on the other -- one barrier per chunk.
//  * The wave computes the transposed products S^T = K . Q^T and O^T = V^T . P^T with
//    v_mfma_f32_16x16x32_bf16, so that every head is one lane column: the online softmax's
//    running max and sum live in the lane, the max and sum over a chunk cross the four
//    16-lane rows with v_permlane32_swap / v_permlane16_swap, and P reaches the B-operand layout
//    of the second product through the same two swaps, without a trip through LDS.
//  * K fragments (8 consecutive dims of one position) come from the staged rows with 16-byte
//    LDS reads, V^T fragments (8 positions of one column) with ds_read_b64_tr_b16, gfx950's
//    transposing LDS read.
//  * Spans write (max, sum, unnormalised output) partials; a merge kernel on the same stream
//    combines them in span order.  From 8 spans on, the head blocks of one span sit on one XCD
//    (workgroup ids 8 apart, the grid padded to whole groups of 8 spans) so the cache rows they
//    share are read from HBM once per XCD.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdlib>

#include "attention_core.h"
#include "bf16_cast.h"
#include "nmm_internal.h"

namespace nmm {
namespace {

using namespace attn;

template <int CH, int KS, int NT, int PMAX, bool EXACT>
__global__ __launch_bounds__(kAThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void attention_kernel(const AttnParams p) {
    attention_block<CH, KS, NT, PMAX, EXACT>(p, blockIdx.x);
}

// Merge the spans of each head in span order:
//   out = sum_s w_s O_s,  w_s = 2^(m_s - M) / sum_q 2^(m_q - M) l_q,  M = max_s m_s.
// One output per thread: a workgroup owns 4 heads x 64 columns, so 64 threads read one
// 256-byte segment of a (head, span) row.  The partial outputs' loads go out first; the spans'
// (max, sum) pairs follow, one pair per thread, into LDS.  Up to 16 spans, wave 0 forms the
// weights with one lane per (span, head) and an xor butterfly across the spans; beyond that one
// thread per head walks them.  The whole merge waits for about one memory round trip.
constexpr int kMergeCols = 64;
constexpr int kMergeHeads = kAThreads / kMergeCols;   // 4
constexpr int kMergeBatch = 32;
constexpr int kMergeMaxSpans = 64;
__global__ __launch_bounds__(kAThreads) void attention_merge_kernel(const AttnParams p) {
    __shared__ float wgt[kMergeMaxSpans * kMergeHeads];      // [span][head of the group]
    __shared__ float mls[kMergeMaxSpans * kMergeHeads * 2];  // [span][head][max, sum]
    const int n_cb = (p.dv + kMergeCols - 1) / kMergeCols;
    const int hq = blockIdx.x / n_cb, cb = blockIdx.x - hq * n_cb;
    const int tid = threadIdx.x;
    const int h0 = hq * kMergeHeads;                      // a multiple of 4: never crosses a head block
    const int hb = h0 / kHB, r0 = h0 - hb * kHB;
    const int i = tid / kMergeCols, n = cb * kMergeCols + (tid % kMergeCols);
    const int h = h0 + i;
    const bool active = h < p.heads && n < p.dv;
    const float* src = p.part_o + (int64_t(hb) * p.nsp * kHB + r0 + i) * p.dv + n;
    const int64_t step = int64_t(kHB) * p.dv;
    float v[kMergeBatch];
#pragma unroll
    for (int u = 0; u < kMergeBatch; ++u) v[u] = (active && u < p.nsp) ? src[u * step] : 0.f;
    for (int t = tid; t < p.nsp * kMergeHeads; t += kAThreads) {
        const int q = t / kMergeHeads, hh = t - q * kMergeHeads;
        const float* ml = p.part_ml + ((int64_t(hb) * p.nsp + q) * kHB + r0 + hh) * 2;
        mls[2 * t] = ml[0];
        mls[2 * t + 1] = ml[1];
    }
    __syncthreads();
    if (p.nsp * kMergeHeads <= 64) {
        // up to 16 spans: lane q * 4 + hh of wave 0 holds span q of head hh; each head's max and
        // normaliser cross the lanes of that head with a fixed xor butterfly (lanes past the
        // spans contribute a weight of 0)
        if (tid < 64) {
            const bool ok = tid < p.nsp * kMergeHeads;
            const float m = ok ? mls[2 * tid] : -INFINITY;
            const float l = ok ? mls[2 * tid + 1] : 0.f;
            float M = m;
#pragma unroll
            for (int off = kMergeHeads; off < 64; off <<= 1) M = fmaxf(M, __shfl_xor(M, off));
            const float w = (m == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m - M);
            float den = w * l;
#pragma unroll
            for (int off = kMergeHeads; off < 64; off <<= 1) den += __shfl_xor(den, off);
            if (ok) wgt[tid] = w * (1.f / den);
        }
    } else if (tid < kMergeHeads) {
        float M = -INFINITY;
        for (int q = 0; q < p.nsp; ++q) M = fmaxf(M, mls[2 * (q * kMergeHeads + tid)]);
        float den = 0.f;
        for (int q = 0; q < p.nsp; ++q) {
            const float mq = mls[2 * (q * kMergeHeads + tid)];
            const float w = (mq == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mq - M);
            den += w * mls[2 * (q * kMergeHeads + tid) + 1];
            wgt[q * kMergeHeads + tid] = w;
        }
        const float inv = 1.f / den;
        for (int q = 0; q < p.nsp; ++q) wgt[q * kMergeHeads + tid] *= inv;
    }
    __syncthreads();
    if (!active) return;
    float acc = 0.f;
    for (int q0 = 0; q0 < p.nsp; q0 += kMergeBatch) {
        if (q0 > 0) {
#pragma unroll
            for (int u = 0; u < kMergeBatch; ++u) v[u] = (q0 + u < p.nsp) ? src[(q0 + u) * step] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u)
            if (q0 + u < p.nsp) acc += wgt[(q0 + u) * kMergeHeads + i] * v[u];
    }
    p.out[int64_t(h) * p.ldo + n] = acc;
    if (p.outb) p.outb[int64_t(h) * p.ldob + n] = to_bf16_bits(acc);
}

struct AttnPlan {
    int n_hb = 0, nsp = 1, span = 0, xcd_map = 0, ch = 64, cols = 0, pitch = 0;
    int grid_sp = 1;    // spans in the grid: nsp, padded to a multiple of 8 when xcd_map
    size_t ws_bytes = 0;
};

int64_t env_splits() {
    const char* s = std::getenv("NMM_ATTN_SPLITS");
    if (!s || !*s) return 0;
    const long long v = std::strtoll(s, nullptr, 10);
    return v > 0 ? v : 0;
}

// splits > 0 asks for that many position spans per head block (the span is rounded up to whole
// chunks, so fewer may result); 0 takes NMM_ATTN_SPLITS or the default of about 64 workgroups.
nmm_status plan_attention(int64_t heads, int64_t seq, int64_t dqk, int64_t dv, AttnPlan* out, int64_t splits = 0) {
    if (heads < 0 || seq < 1 || heads >= (1 << 30) || seq >= (1 << 30)) return NMM_ERR_SHAPE;
    if (dqk < 32 || dqk > 1024 || dqk % 32) return NMM_ERR_SHAPE;
    if (dv < 16 || dv > 512 || dv % 16) return NMM_ERR_SHAPE;
    AttnPlan a;
    a.n_hb = static_cast<int>((heads + kHB - 1) / kHB);
    a.cols = static_cast<int>(std::max(dqk, dv));
    a.pitch = a.cols + 8;
    a.ch = a.cols <= 576 ? 64 : 32;
    if (const char* e = std::getenv("NMM_ATTN_CHUNK"))   // tuning override: 32-position chunks
        if (std::atoi(e) == 32) a.ch = 32;
    const int64_t max_sp = (seq + a.ch - 1) / a.ch;
    int64_t nsp = splits > 0 ? splits : env_splits();
    if (nsp == 0) nsp = std::max<int64_t>(1, 64 / std::max(1, a.n_hb));   // about 64 workgroups
    nsp = std::min(std::min(nsp, max_sp), int64_t(kMergeMaxSpans));
    int64_t span = (seq + nsp - 1) / nsp;
    span = (span + a.ch - 1) / a.ch * a.ch;
    nsp = (seq + span - 1) / span;
    a.nsp = static_cast<int>(nsp);
    a.span = static_cast<int>(span);
    // spans grouped per XCD (the same span of every head block on one XCD, so its cache rows are
    // read once per XCD) from 8 spans on; past 8 the grid is padded to a multiple of 8 spans and
    // the padding workgroups exit at once
    a.xcd_map = (a.nsp % 8 == 0 || a.nsp > 8) ? 1 : 0;
    a.grid_sp = a.xcd_map ? (a.nsp + 7) / 8 * 8 : a.nsp;
    if (a.pitch > (a.ch == 64 ? 584 : 1032)) return NMM_ERR_SHAPE;
    // partial results live past the workspace's counter block (which GEMV calls sharing the
    // workspace rely on being zero)
    if (a.nsp > 1) a.ws_bytes = size_t(kTicketBytes) + size_t(a.n_hb) * a.nsp * kHB * (size_t(dv) + 2) * 4;
    *out = a;
    return NMM_OK;
}

template <int CH, int KS, int NT, int PMAX, bool EXACT>
nmm_status launch_attention(const AttnParams& p, int64_t grid, hipStream_t s) {
    if (p.pitch > PMAX) return NMM_ERR_SHAPE;
    hipLaunchKernelGGL((attention_kernel<CH, KS, NT, PMAX, EXACT>), dim3(static_cast<uint32_t>(grid)), dim3(kAThreads), 0,
                       s, p);
    return hipGetLastError() == hipSuccess ? NMM_OK : NMM_ERR_HIP;
}

}  // namespace
}  // namespace nmm

using namespace nmm;

extern "C" {

size_t nmm_latent_attention_workspace_size(int64_t heads, int64_t seq, int64_t d_qk, int64_t d_v) {
    AttnPlan a;
    return plan_attention(heads, seq, d_qk, d_v, &a) == NMM_OK ? a.ws_bytes : 0;
}

}  // extern "C"

namespace {

// Validation, plan and kernel arguments of one attention call; out->grid stays 0 when there is
// nothing to launch (heads == 0).
nmm_status prepare(int64_t heads, int64_t seq, int64_t d_qk, int64_t d_v, const void* q, int64_t ldq,
                   const void* kv, int64_t ld_kv, float scale, float* out_, int64_t ldo, void* outb,
                   int64_t ldob, int64_t splits, void* workspace, size_t workspace_bytes, AttnLaunch* out) {
    *out = AttnLaunch{};
    if (splits < 0) return NMM_ERR_ARG;
    AttnPlan a;
    nmm_status st = plan_attention(heads, seq, d_qk, d_v, &a, splits);
    if (st != NMM_OK) return st;
    if (!std::isfinite(scale)) return NMM_ERR_ARG;
    if (heads == 0) return NMM_OK;   // nothing to launch (grid 0)
    if (!q || !kv || !out_) return NMM_ERR_NULL;
    if (ldq < d_qk || ld_kv < std::max(d_qk, d_v) || ldo < d_v) return NMM_ERR_SHAPE;
    if (ldq >= (int64_t(1) << 31) || ld_kv >= (int64_t(1) << 31) || ldo >= (int64_t(1) << 31)) return NMM_ERR_SHAPE;
    if ((reinterpret_cast<uintptr_t>(q) & 15u) || (reinterpret_cast<uintptr_t>(kv) & 15u) || ldq % 8 ||
        ld_kv % 8 || (reinterpret_cast<uintptr_t>(out_) & 15u) || ldo % 4)
        return NMM_ERR_ALIGN;
    const int64_t extent = ((seq - 1) * ld_kv + std::max(d_qk, d_v)) * 2;
    const int64_t q_extent = ((heads - 1) * ldq + d_qk) * 2;
    if (extent >= (int64_t(1) << 31) || q_extent >= (int64_t(1) << 31) || ldo >= (int64_t(1) << 31)) return NMM_ERR_SHAPE;
    st = validate_workspace(workspace, workspace_bytes, a.ws_bytes);
    if (st != NMM_OK) return st;

    AttnParams& p = out->p;
    p = AttnParams{};
    p.q = static_cast<const uint16_t*>(q);
    p.ldq = ldq;
    p.kv = static_cast<const uint16_t*>(kv);
    p.ldkv = ld_kv;
    p.out = out_;
    p.ldo = ldo;
    p.outb = static_cast<uint16_t*>(outb);
    p.ldob = ldob;
    if (a.ws_bytes) {
        p.part_o = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + kTicketBytes);
        p.part_ml = p.part_o + size_t(a.n_hb) * a.nsp * kHB * d_v;
    }
    p.heads = static_cast<int>(heads);
    p.seq = static_cast<int>(seq);
    p.dqk = static_cast<int>(d_qk);
    p.dv = static_cast<int>(d_v);
    p.cols = a.cols;
    p.pitch = a.pitch;
    p.nsp = a.nsp;
    p.span = a.span;
    p.n_hb = a.n_hb;
    p.xcd_map = a.xcd_map;
    p.scale_log2 = scale * 1.4426950408889634f;
    p.kv_extent = static_cast<uint32_t>(extent);
    p.q_extent = static_cast<uint32_t>(q_extent);
    out->grid = int64_t(a.n_hb) * a.grid_sp;
    out->merge_grid = a.nsp > 1 ? ((heads + kMergeHeads - 1) / kMergeHeads) * ((d_v + kMergeCols - 1) / kMergeCols) : 0;
    out->variant = (d_qk == 576 && d_v == 512) ? (a.ch == 64 ? kAttnExact64 : kAttnExact32)
                                                : (a.ch == 64 ? kAttnGeneral64 : kAttnGeneral32);
    return NMM_OK;
}

nmm_status attention_common(int64_t heads, int64_t seq, int64_t d_qk, int64_t d_v, const void* q, int64_t ldq,
                            const void* kv, int64_t ld_kv, float scale, float* out, int64_t ldo, void* outb,
                            int64_t ldob, int64_t splits, void* workspace, size_t workspace_bytes, void* stream) {
    AttnLaunch l;
    const nmm_status st = prepare(heads, seq, d_qk, d_v, q, ldq, kv, ld_kv, scale, out, ldo, outb, ldob, splits,
                                  workspace, workspace_bytes, &l);
    if (st != NMM_OK) return st;
    return launch_prepared_attention(l, static_cast<hipStream_t>(stream));
}

}  // namespace

namespace nmm {

nmm_status launch_attention_merge(const AttnLaunch& l, hipStream_t s) {
    if (l.merge_grid == 0) return NMM_OK;
    hipLaunchKernelGGL(attention_merge_kernel, dim3(static_cast<uint32_t>(l.merge_grid)), dim3(kAThreads), 0, s, l.p);
    return hipGetLastError() == hipSuccess ? NMM_OK : NMM_ERR_HIP;
}

nmm_status launch_prepared_attention(const AttnLaunch& l, hipStream_t s) {
    if (l.grid == 0) return NMM_OK;
    nmm_status st;
    switch (l.variant) {
        case kAttnExact64: st = launch_attention<64, 18, 32, 584, true>(l.p, l.grid, s); break;
        case kAttnExact32: st = launch_attention<32, 18, 32, 584, true>(l.p, l.grid, s); break;
        case kAttnGeneral64: st = launch_attention<64, 18, 32, 584, false>(l.p, l.grid, s); break;
        default: st = launch_attention<32, 32, 32, 1032, false>(l.p, l.grid, s); break;
    }
    if (st != NMM_OK) return st;
    return launch_attention_merge(l, s);
}

nmm_status prepare_attention(const AttnArgs& a, void* workspace, size_t workspace_bytes, AttnLaunch* out) {
    if (a.outb && (a.ldob < a.d_v || a.ldob >= (int64_t(1) << 31))) return NMM_ERR_SHAPE;
    if (reinterpret_cast<uintptr_t>(a.outb) & 1u) return NMM_ERR_ALIGN;
    return prepare(a.heads, a.seq, a.d_qk, a.d_v, a.q, a.ldq, a.kv, a.ld_kv, a.scale, a.out, a.ldo, a.outb, a.ldob,
                   a.splits, workspace, workspace_bytes, out);
}

nmm_status attention_workspace_bytes(const AttnArgs& a, size_t* bytes) {
    *bytes = 0;
    if (a.splits < 0) return NMM_ERR_ARG;
    AttnPlan p;
    const nmm_status st = plan_attention(a.heads, a.seq, a.d_qk, a.d_v, &p, a.splits);
    if (st == NMM_OK) *bytes = p.ws_bytes;
    return st;
}

nmm_status validate_attention_args(const AttnArgs& a, void* workspace, size_t workspace_bytes) {
    AttnLaunch l;
    return prepare_attention(a, workspace, workspace_bytes, &l);
}

nmm_status launch_attention_args(const AttnArgs& a, void* workspace, size_t workspace_bytes, void* stream) {
    AttnLaunch l;
    const nmm_status st = prepare_attention(a, workspace, workspace_bytes, &l);
    if (st != NMM_OK) return st;
    return launch_prepared_attention(l, static_cast<hipStream_t>(stream));
}

}  // namespace nmm

extern "C" {

nmm_status nmm_latent_attention(int64_t heads, int64_t seq, int64_t d_qk, int64_t d_v,
                                const void* q, int64_t ldq, const void* kv, int64_t ld_kv,
                                float scale, float* out, int64_t ldo, void* workspace,
                                size_t workspace_bytes, void* stream) {
    return attention_common(heads, seq, d_qk, d_v, q, ldq, kv, ld_kv, scale, out, ldo, nullptr, 0, 0, workspace,
                            workspace_bytes, stream);
}

nmm_status nmm_latent_attention_bf16(int64_t heads, int64_t seq, int64_t d_qk, int64_t d_v,
                                     const void* q, int64_t ldq, const void* kv, int64_t ld_kv,
                                     float scale, float* out, int64_t ldo, void* out_bf16, int64_t ldob,
                                     void* workspace, size_t workspace_bytes, void* stream) {
    if (heads > 0 && !out_bf16) return NMM_ERR_NULL;
    if (ldob < d_v || ldob >= (int64_t(1) << 31)) return NMM_ERR_SHAPE;
    if (reinterpret_cast<uintptr_t>(out_bf16) & 1u) return NMM_ERR_ALIGN;
    return attention_common(heads, seq, d_qk, d_v, q, ldq, kv, ld_kv, scale, out, ldo, out_bf16, ldob, 0, workspace,
                            workspace_bytes, stream);
}

nmm_status nmm_latent_attention_ex(int64_t heads, int64_t seq, int64_t d_qk, int64_t d_v,
                                   const void* q, int64_t ldq, const void* kv, int64_t ld_kv,
                                   float scale, float* out, int64_t ldo, void* out_bf16, int64_t ldob,
                                   int64_t splits, void* workspace, size_t workspace_bytes, void* stream) {
    if (out_bf16 && (ldob < d_v || ldob >= (int64_t(1) << 31))) return NMM_ERR_SHAPE;
    if (reinterpret_cast<uintptr_t>(out_bf16) & 1u) return NMM_ERR_ALIGN;
    return attention_common(heads, seq, d_qk, d_v, q, ldq, kv, ld_kv, scale, out, ldo, out_bf16, ldob, splits,
                            workspace, workspace_bytes, stream);
}

size_t nmm_latent_attention_ex_workspace_size(int64_t heads, int64_t seq, int64_t d_qk, int64_t d_v, int64_t splits) {
    AttnPlan a;
    return splits >= 0 && plan_attention(heads, seq, d_qk, d_v, &a, splits) == NMM_OK ? a.ws_bytes : 0;
}

}  // extern "C"
