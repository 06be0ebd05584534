// Single-token latent attention on the matrix cores (gfx950), the decode step's independent
// dense work.  The paper's point is that narrow MatMuls moved off the matrix unit let
// independent matrix-unit work start earlier (Condition 1 "Data Independence", Section III-A;
// Section IV-A); this kernel is that independent work here, run on its own or with its workgroups
// beside the last narrow MatMul's in one launch (the decode step).
//
//   s_j = scale * q_h . kv_j[:d_qk],  p = softmax(s),  out_h = sum_j p_j kv_j[:d_v]
//
// Every head reads the same latent cache, so the work is two dense products per span of
// positions, S = Q . K^T and O = P . V, with a softmax between them (flash-decoding):
//  * A workgroup owns a block of heads and a span of positions, walked in 64-position chunks.  A
//    chunk's rows (the first max(d_qk, d_v) columns) are staged in LDS by buffer loads that write
//    LDS directly, into one of two buffers while the waves compute on the other.  This launch
//    takes blocks of 16 heads (one 16-head MFMA tile); workgroups that share a launch with a GEMV
//    take 32 heads (two tiles), and so does this launch when such a call cannot share one.  Every
//    workgroup has 4 waves, one per SIMD, each taking all of the block's head tiles.
//  * Q.K^T is split by positions: position group w % 4 computes S^T = K . Q^T for positions
//    16 (w % 4) .. + 15 of the chunk (v_mfma_f32_16x16x32_bf16; Q sits in registers as MFMA
//    fragments) for the wave's head tiles, each K fragment read from LDS feeding every tile's MFMA.
//  * The softmax reference of a head is the running maximum, moved only when a chunk exceeds it
//    by more than 2^8 (then the output is rescaled, rarely): P = 2^(s - reference) is rounded to
//    bf16 and exchanged through LDS.  The chunk maxima cross the waves through LDS as well.
//  * P.V is split by output columns: position group w % 4 accumulates O^T = V^T . P^T for the
//    16-column tiles w % 4, w % 4 + 4, ... of its heads, V^T fragments read from the staged rows
//    by ds_read_b64_tr_b16 (gfx950's transposing LDS read).  The accumulators stay in registers.
//    At 576 / 512, while the grid fits one workgroup per CU, four or two workgroups share each
//    (head block, span), each taking its share of the column tiles (all compute the scores):
//    more workgroups, each with a share of the P.V work and the stores.
//  * Spans write (reference, sum, unnormalised output) partials; a merge kernel on the same
//    stream combines them in span order.  The head blocks of one span run on one XCD (workgroup
//    ids 8 apart), so its L2 reads the span's cache rows from HBM once for all of them.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "attention_core.h"
#include "bf16_cast.h"
#include "nmm_internal.h"

namespace nmm {
namespace {

using namespace attn;

// Heads per workgroup.  The attention launch takes blocks of 16 (one head tile, 4 waves, one per
// SIMD): twice the workgroups of 32-head blocks over the same spans, each with half the matrix work
// per staged chunk.  Workgroups that share a launch with a GEMV take 32 (two head tiles, 4 waves),
// so that they hold half as many compute units beside the GEMV's weight stream.  No head's
// arithmetic depends on which heads share its block, so the two give the same bits.
constexpr int kAloneHeads = 16;
constexpr int kSharedHeads = 16 * kHt;   // 32
constexpr int kMaxSpans = 64;             // the merge gives each span one lane of a wave
constexpr int kDefaultPairs = 64;         // default partition: about this many (32-head block, span) pairs,
constexpr int kDefaultMaxChunks = 8;      // or more spans, so that a span has at most about this many chunks,
constexpr int kDefaultFitChunks = 4;      // or this many while one workgroup per 16-head block and span fits the CUs,
constexpr int kDefaultMinChunks = 2;      // but spans of at least this many chunks (one-chunk spans merge
                                          // more partials than their parallelism saves)
constexpr int kComputeUnits = 256;        // MI355X; an attention workgroup holds a CU (its LDS)

// Attention launch workgroups of HT head tiles, each taking 4 NTW of d_v's 16-column tiles (of
// VS column parts).
template <int HT, int NTW, bool EXACT, int VS>
__global__ __launch_bounds__(kAThreads) void attention_kernel(const AttnParams p) {
    attention_block<HT, kMaxKs, NTW, EXACT, VS>(p, blockIdx.x);
}

__global__ __launch_bounds__(kMergeWideThreads) void attention_merge_kernel(const AttnParams p) {
    merge_block_wide(p, static_cast<int>(blockIdx.x));
}

struct AttnPlan {
    int hbh = kAloneHeads;
    int vsplit = 1;     // workgroups per (head block, span)
    int n_hb = 0, nsp = 1, span = 0, xcd_map = 0, cols = 0, pitch = 0;
    int grid_sp = 1;    // spans in the grid: nsp, padded to a multiple of 8 when xcd_map
    size_t ws_bytes = 0;
};

// splits > 0 asks for that many position spans (the span is rounded up to whole chunks, so fewer
// may result); 0 takes the default.  The spans do not depend on the head block (16 or 32 heads),
// and the workspace is sized for 32-head blocks, which covers both.  hbh == kAloneHeads asks for
// 16-head blocks, which the plan widens to 32 heads when their grid would take more than one
// round of the CUs (every head's arithmetic is the same in either block, so the results are too).
nmm_status plan_attention(int64_t heads, int64_t seq, int64_t dqk, int64_t dv, AttnPlan* out, int64_t splits = 0,
                          int hbh = kAloneHeads) {
    if (heads < 0 || seq < 1 || heads >= (1 << 30) || seq >= (1 << 30)) return NMM_ERR_SHAPE;
    if (dqk < 32 || dqk > kMaxCols || dqk % 32) return NMM_ERR_SHAPE;
    if (dv < 16 || dv > 16 * 4 * kMaxNtw || dv % 16) return NMM_ERR_SHAPE;
    if (splits < 0) return NMM_ERR_ARG;
    AttnPlan a;
    a.hbh = hbh;
    a.n_hb = static_cast<int>((heads + hbh - 1) / hbh);
    a.cols = static_cast<int>(std::max(dqk, dv));
    a.pitch = a.cols + 8 * kPadSlots;
    const int64_t wide_blocks = (heads + kSharedHeads - 1) / kSharedHeads;
    const int64_t max_sp = (seq + kCh - 1) / kCh;
    const int64_t few_chunk_spans = (seq + kDefaultMinChunks * kCh - 1) / (kDefaultMinChunks * kCh);
    const int64_t short_spans = (seq + kDefaultMaxChunks * kCh - 1) / (kDefaultMaxChunks * kCh);
    // rounded down, so that a ragged tail (4097 positions) keeps spans of more than four chunks
    const int64_t shorter_spans = std::max<int64_t>(1, max_sp / kDefaultFitChunks);
    const int64_t pair_spans = kDefaultPairs / std::max<int64_t>(1, wide_blocks);
    // spans that a grid of 16-head blocks holds at one workgroup per CU (a multiple of 8 from 8 on,
    // so the XCD-grouped grid needs no padding)
    int64_t fit_spans = kComputeUnits / std::max<int64_t>(1, (heads + kAloneHeads - 1) / kAloneHeads);
    if (fit_spans >= 8) fit_spans = fit_spans / 8 * 8;
    const int64_t want = std::max(std::max(pair_spans, short_spans), std::min(shorter_spans, fit_spans));
    int64_t nsp = splits > 0 ? splits : std::max<int64_t>(1, std::min(few_chunk_spans, want));
    nsp = std::min(std::min(nsp, max_sp), int64_t(kMaxSpans));
    int64_t span = (seq + nsp - 1) / nsp;
    span = (span + kCh - 1) / kCh * kCh;
    nsp = (seq + span - 1) / span;
    a.nsp = static_cast<int>(nsp);
    a.span = static_cast<int>(span);
    // from 8 spans on, the head blocks of a span share an XCD (ids 8 apart); past a multiple of 8
    // the grid is padded and the padding workgroups exit at once
    a.xcd_map = (a.nsp % 8 == 0 || a.nsp > 8) ? 1 : 0;
    a.grid_sp = a.xcd_map ? (a.nsp + 7) / 8 * 8 : a.nsp;
    // past one workgroup per CU, 32-head blocks halve the grid (and the K / V chunk reads) rather
    // than running the 16-head grid in two rounds
    if (hbh == kAloneHeads && heads > kAloneHeads && int64_t(a.n_hb) * a.grid_sp > kComputeUnits) {
        a.hbh = kSharedHeads;
        a.n_hb = static_cast<int>(wide_blocks);
    }
    // the 576 / 512 shape in 16-head blocks splits d_v over four or two workgroups per (head
    // block, span) while the grid still fits one workgroup per CU
    if (a.hbh == kAloneHeads && dqk == kMaxCols && dv == 16 * 4 * kMaxNtw) {
        if (int64_t(a.n_hb) * 4 * a.grid_sp <= kComputeUnits) a.vsplit = 4;
        else if (int64_t(a.n_hb) * 2 * a.grid_sp <= kComputeUnits) a.vsplit = 2;
    }
    // partial results live past the workspace's counter block (which GEMV calls sharing the
    // workspace rely on being zero)
    if (a.nsp > 1)
        a.ws_bytes = size_t(kTicketBytes) + size_t(wide_blocks) * kSharedHeads * a.nsp * (size_t(dv) + 2) * 4;
    *out = a;
    return NMM_OK;
}

template <bool EXACT>
nmm_status launch_attention(const AttnParams& p, int64_t grid, int vsplit, hipStream_t s) {
    const dim3 g(static_cast<uint32_t>(grid));
    if (vsplit == 4)
        hipLaunchKernelGGL((attention_kernel<1, kMaxNtw / 4, true, 4>), g, dim3(kAThreads), 0, s, p);
    else if (vsplit == 2)
        hipLaunchKernelGGL((attention_kernel<1, kMaxNtw / 2, true, 2>), g, dim3(kAThreads), 0, s, p);
    else if (p.hbh == kAloneHeads)
        hipLaunchKernelGGL((attention_kernel<1, kMaxNtw, EXACT, 1>), g, dim3(kAThreads), 0, s, p);
    else
        hipLaunchKernelGGL((attention_kernel<kHt, kMaxNtw, EXACT, 1>), g, dim3(kAThreads), 0, s, p);
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

// Validation, plan and kernel arguments of one attention call in blocks of hbh heads; out->grid
// stays 0 when there is nothing to launch (heads == 0).
nmm_status prepare(int64_t heads, int64_t seq, int64_t d_qk, int64_t d_v, const void* q, int64_t ldq,
                   const void* kv, int64_t ld_kv, float scale, float* out_, int64_t ldo, void* outb,
                   int64_t ldob, int64_t splits, void* workspace, size_t workspace_bytes, int hbh, AttnLaunch* out) {
    *out = AttnLaunch{};
    if (splits < 0) return NMM_ERR_ARG;
    AttnPlan a;
    nmm_status st = plan_attention(heads, seq, d_qk, d_v, &a, splits, hbh);
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
    if (extent >= (int64_t(1) << 31) || q_extent >= (int64_t(1) << 31)) return NMM_ERR_SHAPE;
    // a chunk's row offsets (up to kCh rows past the last one) are 32-bit
    if ((seq + kCh) * ld_kv * 2 >= (int64_t(1) << 32)) return NMM_ERR_SHAPE;
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
        p.part_ml = p.part_o + size_t(a.n_hb) * a.nsp * a.hbh * d_v;
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
    p.hbh = a.hbh;
    p.xcd_map = a.xcd_map;
    p.scale_log2 = scale * 1.4426950408889634f;
    p.kv_extent = static_cast<uint32_t>(extent);
    p.q_extent = static_cast<uint32_t>(q_extent);
    out->grid = int64_t(a.n_hb) * a.vsplit * a.grid_sp;
    out->merge_grid = a.nsp > 1 ? heads * ((d_v + kMergeThreads - 1) / kMergeThreads) : 0;
    out->variant = (d_qk == 576 && d_v == 512) ? kAttnExact : kAttnGeneral;
    out->vsplit = a.vsplit;
    return NMM_OK;
}

nmm_status attention_common(int64_t heads, int64_t seq, int64_t d_qk, int64_t d_v, const void* q, int64_t ldq,
                            const void* kv, int64_t ld_kv, float scale, float* out, int64_t ldo, void* outb,
                            int64_t ldob, int64_t splits, void* workspace, size_t workspace_bytes, void* stream) {
    AttnLaunch l;
    const nmm_status st = prepare(heads, seq, d_qk, d_v, q, ldq, kv, ld_kv, scale, out, ldo, outb, ldob, splits,
                                  workspace, workspace_bytes, kAloneHeads, &l);
    if (st != NMM_OK) return st;
    return launch_prepared_attention(l, static_cast<hipStream_t>(stream));
}

}  // namespace

namespace nmm {

nmm_status launch_attention_merge(const AttnLaunch& l, hipStream_t s) {
    if (l.merge_grid == 0) return NMM_OK;
    static_assert(4 * kMergeWideThreads == kMergeThreads, "the two merge forms cut a head's columns alike");
    hipLaunchKernelGGL(attention_merge_kernel, dim3(static_cast<uint32_t>(l.merge_grid)), dim3(kMergeWideThreads), 0,
                       s, l.p);
    return hipGetLastError() == hipSuccess ? NMM_OK : NMM_ERR_HIP;
}

nmm_status launch_attention_kernel(const AttnLaunch& l, hipStream_t s) {
    if (l.grid == 0) return NMM_OK;
    return l.variant == kAttnExact ? launch_attention<true>(l.p, l.grid, l.vsplit, s)
                                   : launch_attention<false>(l.p, l.grid, l.vsplit, s);
}

nmm_status launch_prepared_attention(const AttnLaunch& l, hipStream_t s) {
    const nmm_status st = launch_attention_kernel(l, s);
    if (st != NMM_OK) return st;
    return launch_attention_merge(l, s);
}

nmm_status prepare_attention(const AttnArgs& a, void* workspace, size_t workspace_bytes, AttnLaunch* out) {
    if (a.outb && (a.ldob < a.d_v || a.ldob >= (int64_t(1) << 31))) return NMM_ERR_SHAPE;
    if (reinterpret_cast<uintptr_t>(a.outb) & 1u) return NMM_ERR_ALIGN;
    return prepare(a.heads, a.seq, a.d_qk, a.d_v, a.q, a.ldq, a.kv, a.ld_kv, a.scale, a.out, a.ldo, a.outb, a.ldob,
                   a.splits, workspace, workspace_bytes, kSharedHeads, out);
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
