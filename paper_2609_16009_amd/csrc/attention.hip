// Single-token latent attention on the matrix cores (gfx950), the decode step's independent
// dense work.  The paper's point is that narrow MatMuls moved off the matrix unit let
// independent matrix-unit work start earlier (Condition 1 "Data Independence", Section III-A;
// Section IV-A); this kernel is that independent work here, run on its own stream.
//
//   s_j = scale * q_h . kv_j[:d_qk],  p = softmax(s),  out_h = sum_j p_j kv_j[:d_v]
//
// Design (flash-decoding):
//  * A workgroup owns 16 heads (one MFMA row tile) and a contiguous span of positions.  It keeps
//    Q's 16 rows in LDS and walks its span in chunks of 64 positions with an online softmax.
//  * QK^T: each of the 4 waves scores 16 positions with v_mfma_f32_16x16x32_bf16; Q fragments
//    come from LDS, K fragments straight from global memory (a lane's 8 k-values are one
//    contiguous 16-byte piece of a cache row).
//  * Chunk maxima and sums cross waves through LDS; P is rounded to bf16 into LDS.
//  * P.V: wave w owns the output column tiles w, w+4, ...; V is staged through LDS row-major and
//    read back with ds_read_b64_tr_b16, gfx950's transposing LDS read, which hands each lane the
//    8 positions of one column that the MFMA B operand needs.
//  * Every load of the next chunk (K fragments, both halves of V) is issued one chunk ahead,
//    branch-free: positions outside the span read zeros through the buffer's range check.
//  * The spans' partial (max, sum, output) go to the workspace; a small merge kernel on the same
//    stream combines them in span order (the kernel boundary makes the partials visible).
//  * Workgroups of one span are placed on the same XCD (ids 8 apart) so the span's K/V rows are
//    read from HBM once per XCD and then served from that XCD's L2.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "nmm_internal.h"

namespace nmm {
namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr int kAHeads = 16;       // heads per workgroup
constexpr int kAChunk = 64;       // positions per chunk (16 per wave)
constexpr int kAThreads = 256;
constexpr int kAMaxTiles = 8;     // output column tiles per wave (d_v <= 512)
constexpr int kRsrcWord3 = 0x00020000;
constexpr uint32_t kOutOfRange = 0x80000000u;

struct AttnParams {
    const uint16_t* q;
    int64_t ldq;
    const uint16_t* kv;
    int64_t ldkv;
    float* out;
    int64_t ldo;
    float* part_o;      // [n_hb][nsp][16][d_v]
    float* part_ml;     // [n_hb][nsp][16][2]
    int heads, seq, dqk, dv;
    int nsp, span, n_hb;
    int xcd_map;        // 1: spans grouped per XCD (nsp % 8 == 0)
    float scale_log2;   // scale * log2(e): scores are kept in log2 units
    uint32_t kv_extent; // bytes of the cache that may be read
    int q_stride;       // LDS row stride of Q (elements)
    int v_stride;       // LDS row stride of V (elements)
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kRsrcWord3);
}

__device__ __forceinline__ bf16x8 as_bf16x8(i32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ float row16_max(float v) {
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ __forceinline__ float row16_sum(float v) {
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ __forceinline__ uint16_t bf16_bits(float v) {
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(v));
}

// One chunk's K fragments for this lane: position `pos`, 8 dims per MFMA k-step.
template <int KS>
__device__ __forceinline__ void load_k(i32x4 (&kb)[KS], __amdgpu_buffer_rsrc_t kvr, int pos, bool ok,
                                       int64_t ldkv, int g, int ksteps) {
    const uint32_t base = uint32_t((int64_t(pos) * ldkv + 8 * g) * 2);
#pragma unroll
    for (int u = 0; u < KS; ++u)
        kb[u] = __builtin_amdgcn_raw_buffer_load_b128(kvr, (ok && u < ksteps) ? base + u * 64 : kOutOfRange, 0, 0);
}

// One half chunk (32 positions) of V rows, this thread's 16-byte pieces.
template <int VP>
__device__ __forceinline__ void load_v(i32x4 (&vr)[VP], __amdgpu_buffer_rsrc_t kvr, int r0, int s_end,
                                       int64_t ldkv, int vchunks, int tid) {
#pragma unroll
    for (int q = 0; q < VP; ++q) {
        const int i = tid + q * kAThreads;
        const int r = i / vchunks, c = i - r * vchunks;
        const bool ok = i < 32 * vchunks && r0 + r < s_end;
        vr[q] = __builtin_amdgcn_raw_buffer_load_b128(kvr, ok ? uint32_t((int64_t(r0 + r) * ldkv + 8 * c) * 2) : kOutOfRange,
                                                      0, 0);
    }
}

template <int VP>
__device__ __forceinline__ void store_v(const i32x4 (&vr)[VP], uint16_t* v_lds, int v_stride, int vchunks, int tid) {
#pragma unroll
    for (int q = 0; q < VP; ++q) {
        const int i = tid + q * kAThreads;
        if (i < 32 * vchunks) {
            const int r = i / vchunks, c = i - r * vchunks;
            *reinterpret_cast<i32x4*>(v_lds + r * v_stride + 8 * c) = vr[q];
        }
    }
}

// The span's partial result for 16 heads: running max (log2 units), running sum, and the
// unnormalised output, all written with plain stores; the merge kernel, launched next on the
// same stream, reads them.
template <int KS, int VP, int QP>
__global__ __launch_bounds__(kAThreads) void attention_kernel(const AttnParams p) {
    extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
    __shared__ float red_max[4][kAHeads];
    __shared__ float red_sum[4][kAHeads];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, j = lane & 15;

    int hb, sp;
    const int bid = blockIdx.x;
    if (p.xcd_map) {
        sp = (bid & 7) + 8 * (bid / (8 * p.n_hb));
        hb = (bid >> 3) % p.n_hb;
    } else {
        hb = bid % p.n_hb;
        sp = bid / p.n_hb;
    }
    const int h0 = hb * kAHeads;
    const int s_begin = sp * p.span;
    const int s_end = min(p.seq, s_begin + p.span);

    uint16_t* q_lds = smem;                                    // [16][q_stride]
    uint16_t* p_lds = q_lds + kAHeads * p.q_stride;            // [16][72]
    uint16_t* v_lds = p_lds + kAHeads * (kAChunk + 8);         // [32][v_stride]
    constexpr int kPStride = kAChunk + 8;

    const __amdgpu_buffer_rsrc_t kvr = make_rsrc(p.kv, p.kv_extent);
    const int ksteps = p.dqk / 32;
    const int vchunks = p.dv / 8;
    // ---- Q block: every load issued at once (rows past `heads` read zeros), then the first
    // chunk's K and V loads, then Q goes to LDS while those are in flight
    const int qcpr = p.dqk / 8;
    i32x4 qv[QP];
    {
        const int64_t q_rows = min(kAHeads, p.heads - h0);
        const __amdgpu_buffer_rsrc_t qr =
            make_rsrc(p.q + int64_t(h0) * p.ldq, uint32_t(((q_rows - 1) * p.ldq + p.dqk) * 2));
#pragma unroll
        for (int u = 0; u < QP; ++u) {
            const int i = tid + u * kAThreads;
            const int r = i / qcpr, c = i - r * qcpr;
            const bool ok = i < kAHeads * qcpr && r < q_rows;
            qv[u] = __builtin_amdgcn_raw_buffer_load_b128(qr, ok ? uint32_t((int64_t(r) * p.ldq + 8 * c) * 2) : kOutOfRange,
                                                          0, 0);
        }
    }
    i32x4 kb[KS], v0[VP], v1[VP];
    load_k<KS>(kb, kvr, s_begin + 16 * wave + j, s_begin + 16 * wave + j < s_end, p.ldkv, g, ksteps);
    load_v<VP>(v0, kvr, s_begin, s_end, p.ldkv, vchunks, tid);
    load_v<VP>(v1, kvr, s_begin + 32, s_end, p.ldkv, vchunks, tid);
#pragma unroll
    for (int u = 0; u < QP; ++u) {
        const int i = tid + u * kAThreads;
        if (i < kAHeads * qcpr) {
            const int r = i / qcpr, c = i - r * qcpr;
            *reinterpret_cast<i32x4*>(q_lds + r * p.q_stride + 8 * c) = qv[u];
        }
    }
    const int ntiles = p.dv / 16;
    const int my_tiles = (ntiles - wave + 3) / 4;              // tiles w, w+4, ...
    f32x4 o[kAMaxTiles];
#pragma unroll
    for (int t = 0; t < kAMaxTiles; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run[4], l_run[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        m_run[i] = -INFINITY;
        l_run[i] = 0.f;
    }
    __syncthreads();

    for (int c0 = s_begin; c0 < s_end; c0 += kAChunk) {
        const int next = c0 + kAChunk;
        // ---- scores for this wave's 16 positions: S[16 heads][16 pos] = Q . K^T
        const int pos = c0 + 16 * wave + j;
        const bool pos_ok = pos < s_end;
        f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f}, s2 = f32x4{0.f, 0.f, 0.f, 0.f};   // two chains
#pragma unroll
        for (int u = 0; u < KS; ++u) {
            if (u < ksteps) {
                const i32x4 a = *reinterpret_cast<const i32x4*>(q_lds + j * p.q_stride + 32 * u + 8 * g);
                if (u & 1) s2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(kb[u]), s2, 0, 0, 0);
                else s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(kb[u]), s, 0, 0, 0);
            }
        }
        s += s2;
        // next chunk's K fragments fly during the softmax and P.V below
        load_k<KS>(kb, kvr, next + 16 * wave + j, next + 16 * wave + j < s_end, p.ldkv, g, ksteps);

        // scores in log2 units: s * scale * log2(e), so softmax weights are exp2(s - max)
#pragma unroll
        for (int i = 0; i < 4; ++i) s[i] = pos_ok ? s[i] * p.scale_log2 : -INFINITY;
        float cm[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) cm[i] = row16_max(s[i]);
        if (j == 0) {
#pragma unroll
            for (int i = 0; i < 4; ++i) red_max[wave][4 * g + i] = cm[i];
        }
        __syncthreads();
        float m_new[4], alpha[4], pr[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = 4 * g + i;
            const float mc = fmaxf(fmaxf(red_max[0][r], red_max[1][r]), fmaxf(red_max[2][r], red_max[3][r]));
            m_new[i] = fmaxf(m_run[i], mc);
            alpha[i] = (m_run[i] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_run[i] - m_new[i]);
            pr[i] = pos_ok ? __builtin_amdgcn_exp2f(s[i] - m_new[i]) : 0.f;
            p_lds[r * kPStride + 16 * wave + j] = bf16_bits(pr[i]);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float cs = row16_sum(pr[i]);
            if (j == 0) red_sum[wave][4 * g + i] = cs;
        }
        store_v<VP>(v0, v_lds, p.v_stride, vchunks, tid);      // V rows c0 .. c0+31
        __syncthreads();
        load_v<VP>(v0, kvr, next, s_end, p.ldkv, vchunks, tid);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = 4 * g + i;
            l_run[i] = alpha[i] * l_run[i] + ((red_sum[0][r] + red_sum[1][r]) + (red_sum[2][r] + red_sum[3][r]));
            m_run[i] = m_new[i];
        }
#pragma unroll
        for (int t = 0; t < kAMaxTiles; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) o[t][i] *= alpha[i];

        // ---- P . V in two halves of 32 positions (one MFMA k-step each)
        const int a4 = j >> 2, b4 = j & 3;
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            if (half == 1) {
                __syncthreads();                                  // every wave is done with half 0
                store_v<VP>(v1, v_lds, p.v_stride, vchunks, tid);  // V rows c0+32 .. c0+63
                __syncthreads();
                load_v<VP>(v1, kvr, next + 32, s_end, p.ldkv, vchunks, tid);
            }
            const i32x4 a = *reinterpret_cast<const i32x4*>(p_lds + j * kPStride + 32 * half + 8 * g);
#pragma unroll
            for (int t = 0; t < kAMaxTiles; ++t) {
                if (t < my_tiles) {
                    const int n0 = 16 * (wave + 4 * t);
                    const uint16_t* base = v_lds + (8 * g + a4) * p.v_stride + n0 + 4 * b4;
                    const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(base));
                    const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(base + 4 * p.v_stride));
                    const uint2 ulo = __builtin_bit_cast(uint2, lo), uhi = __builtin_bit_cast(uint2, hi);
                    const i32x4 b = i32x4{int(ulo.x), int(ulo.y), int(uhi.x), int(uhi.y)};
                    o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), o[t], 0, 0, 0);
                }
            }
        }
        __syncthreads();   // P, V and the reductions are reused by the next chunk
    }

    // ---- this span's result
    if (p.nsp == 1) {
#pragma unroll
        for (int t = 0; t < kAMaxTiles; ++t) {
            if (t < my_tiles) {
                const int n = 16 * (wave + 4 * t) + j;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int h = h0 + 4 * g + i;
                    if (h < p.heads) p.out[int64_t(h) * p.ldo + n] = o[t][i] / l_run[i];
                }
            }
        }
        return;
    }
    const int64_t pidx = int64_t(hb) * p.nsp + sp;
    float* po = p.part_o + pidx * (kAHeads * int64_t(p.dv));
#pragma unroll
    for (int t = 0; t < kAMaxTiles; ++t) {
        if (t < my_tiles) {
            const int n = 16 * (wave + 4 * t) + j;
#pragma unroll
            for (int i = 0; i < 4; ++i) po[(4 * g + i) * p.dv + n] = o[t][i];
        }
    }
    if (wave == 0 && j == 0) {
        float* pml = p.part_ml + pidx * (kAHeads * 2);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            pml[(4 * g + i) * 2] = m_run[i];
            pml[(4 * g + i) * 2 + 1] = l_run[i];
        }
    }
}

// Merge the spans of each head block in span order:
//   out = sum_s w_s O_s,  w_s = 2^(m_s - M) / sum_q 2^(m_q - M) l_q,  M = max_s m_s.
// One workgroup per (head block, 16 output columns): thread (r, c) owns head r, column c and
// issues the loads of all its spans at once.
constexpr int kMergeCols = 16;
__global__ __launch_bounds__(kAThreads) void attention_merge_kernel(const AttnParams p) {
    extern __shared__ __attribute__((aligned(16))) float mls[];   // [nsp][16][2], then [16][nsp]
    float* wgt = mls + p.nsp * kAHeads * 2;
    const int n_cb = (p.dv + kMergeCols - 1) / kMergeCols;
    const int hb = blockIdx.x / n_cb, cb = blockIdx.x - hb * n_cb;
    const int h0 = hb * kAHeads;
    const int tid = threadIdx.x;
    const float* ml = p.part_ml + int64_t(hb) * p.nsp * (kAHeads * 2);
    for (int i = tid; i < p.nsp * kAHeads * 2; i += kAThreads) mls[i] = ml[i];
    __syncthreads();
    if (tid < kAHeads) {
        const int r = tid;
        float M = -INFINITY;
        for (int q = 0; q < p.nsp; ++q) M = fmaxf(M, mls[(q * kAHeads + r) * 2]);
        float den = 0.f;
        for (int q = 0; q < p.nsp; ++q) {
            const float mq = mls[(q * kAHeads + r) * 2];
            const float w = (mq == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mq - M);
            wgt[r * p.nsp + q] = w;
            den += w * mls[(q * kAHeads + r) * 2 + 1];
        }
        for (int q = 0; q < p.nsp; ++q) wgt[r * p.nsp + q] /= den;
    }
    __syncthreads();
    const int r = tid / kMergeCols, n = cb * kMergeCols + (tid % kMergeCols);
    if (h0 + r >= p.heads || n >= p.dv) return;
    const float* src = p.part_o + int64_t(hb) * p.nsp * (kAHeads * int64_t(p.dv)) + r * p.dv + n;
    float acc = 0.f;
    for (int q0 = 0; q0 < p.nsp; q0 += 16) {
        float v[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) v[u] = (q0 + u < p.nsp) ? src[int64_t(q0 + u) * (kAHeads * p.dv)] : 0.f;
#pragma unroll
        for (int u = 0; u < 16; ++u)
            if (q0 + u < p.nsp) acc += wgt[r * p.nsp + q0 + u] * v[u];
    }
    p.out[int64_t(h0 + r) * p.ldo + n] = acc;
}

struct AttnPlan {
    int n_hb = 0, nsp = 1, span = 0, xcd_map = 0;
    size_t ws_bytes = 0;
    size_t lds_bytes = 0, merge_lds_bytes = 0;
    int q_stride = 0, v_stride = 0;
};

int64_t env_splits() {
    const char* s = std::getenv("NMM_ATTN_SPLITS");
    if (!s || !*s) return 0;
    const long long v = std::strtoll(s, nullptr, 10);
    return v > 0 ? v : 0;
}

nmm_status plan_attention(int64_t heads, int64_t seq, int64_t dqk, int64_t dv, AttnPlan* out) {
    if (heads < 0 || seq < 1 || heads >= (1 << 30) || seq >= (1 << 30)) return NMM_ERR_SHAPE;
    if (dqk < 32 || dqk > 1024 || dqk % 32) return NMM_ERR_SHAPE;
    if (dv < 16 || dv > 16 * 4 * kAMaxTiles || dv % 16) return NMM_ERR_SHAPE;
    AttnPlan a;
    a.n_hb = static_cast<int>((heads + kAHeads - 1) / kAHeads);
    const int64_t max_sp = (seq + kAChunk - 1) / kAChunk;
    int64_t nsp = env_splits();
    if (nsp == 0) nsp = std::max<int64_t>(1, 128 / std::max(1, a.n_hb));   // about 128 workgroups
    nsp = std::min(nsp, max_sp);
    int64_t span = (seq + nsp - 1) / nsp;
    span = (span + kAChunk - 1) / kAChunk * kAChunk;
    nsp = (seq + span - 1) / span;
    a.nsp = static_cast<int>(nsp);
    a.span = static_cast<int>(span);
    a.xcd_map = (a.nsp % 8 == 0) ? 1 : 0;
    a.q_stride = static_cast<int>(dqk) + 8;
    a.v_stride = static_cast<int>(dv) + 8;
    a.lds_bytes = size_t(kAHeads * a.q_stride + kAHeads * (kAChunk + 8) + 32 * a.v_stride) * 2;
    a.merge_lds_bytes = size_t(kAHeads) * a.nsp * 3 * 4;
    if (a.lds_bytes > 64 * 1024 || a.merge_lds_bytes > 64 * 1024) return NMM_ERR_SHAPE;
    // partial results live past the workspace's counter block (which GEMV calls sharing the
    // workspace rely on being zero)
    if (a.nsp > 1) a.ws_bytes = size_t(kTicketBytes) + size_t(a.n_hb) * a.nsp * kAHeads * (size_t(dv) + 2) * 4;
    *out = a;
    return NMM_OK;
}

}  // namespace
}  // namespace nmm

using namespace nmm;

extern "C" {

size_t nmm_latent_attention_workspace_size(int64_t heads, int64_t seq, int64_t d_qk, int64_t d_v) {
    AttnPlan a;
    return plan_attention(heads, seq, d_qk, d_v, &a) == NMM_OK ? a.ws_bytes : 0;
}

nmm_status nmm_latent_attention(int64_t heads, int64_t seq, int64_t d_qk, int64_t d_v,
                                const void* q, int64_t ldq, const void* kv, int64_t ld_kv,
                                float scale, float* out, int64_t ldo, void* workspace,
                                size_t workspace_bytes, void* stream) {
    AttnPlan a;
    nmm_status st = plan_attention(heads, seq, d_qk, d_v, &a);
    if (st != NMM_OK) return st;
    if (!std::isfinite(scale)) return NMM_ERR_ARG;
    if (heads == 0) return NMM_OK;
    if (!q || !kv || !out) return NMM_ERR_NULL;
    if (ldq < d_qk || ld_kv < std::max(d_qk, d_v) || ldo < d_v) return NMM_ERR_SHAPE;
    if ((reinterpret_cast<uintptr_t>(q) & 15u) || (reinterpret_cast<uintptr_t>(kv) & 15u) || ldq % 8 ||
        ld_kv % 8 || (reinterpret_cast<uintptr_t>(out) & 3u))
        return NMM_ERR_ALIGN;
    const int64_t extent = ((seq - 1) * ld_kv + std::max(d_qk, d_v)) * 2;
    if (extent >= (int64_t(1) << 31) || ldq >= (int64_t(1) << 31) || ldo >= (int64_t(1) << 31)) return NMM_ERR_SHAPE;
    st = validate_workspace(workspace, workspace_bytes, a.ws_bytes);
    if (st != NMM_OK) return st;

    AttnParams p{};
    p.q = static_cast<const uint16_t*>(q);
    p.ldq = ldq;
    p.kv = static_cast<const uint16_t*>(kv);
    p.ldkv = ld_kv;
    p.out = out;
    p.ldo = ldo;
    if (a.ws_bytes) {
        p.part_o = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + kTicketBytes);
        p.part_ml = p.part_o + size_t(a.n_hb) * a.nsp * kAHeads * d_v;
    }
    p.heads = static_cast<int>(heads);
    p.seq = static_cast<int>(seq);
    p.dqk = static_cast<int>(d_qk);
    p.dv = static_cast<int>(d_v);
    p.nsp = a.nsp;
    p.span = a.span;
    p.n_hb = a.n_hb;
    p.xcd_map = a.xcd_map;
    p.scale_log2 = scale * 1.4426950408889634f;
    p.kv_extent = static_cast<uint32_t>(extent);
    p.q_stride = a.q_stride;
    p.v_stride = a.v_stride;
    const int64_t grid = int64_t(a.n_hb) * a.nsp;
    hipStream_t s = static_cast<hipStream_t>(stream);
    // K fragments per lane (d_qk / 32, up to 32) and V pieces per thread per half chunk
    const int ks = static_cast<int>(d_qk / 32);
    const int vp = static_cast<int>((32 * (d_v / 8) + kAThreads - 1) / kAThreads);
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, dim3(static_cast<uint32_t>(grid)), dim3(kAThreads), a.lds_bytes, s, p);
    };
    const int qp = static_cast<int>((kAHeads * (d_qk / 8) + kAThreads - 1) / kAThreads);
    if (ks <= 18 && vp <= 8 && qp <= 5) go(attention_kernel<18, 8, 5>);
    else if (ks <= 32 && vp <= 8 && qp <= 8) go(attention_kernel<32, 8, 8>);
    else return NMM_ERR_SHAPE;
    if (hipGetLastError() != hipSuccess) return NMM_ERR_HIP;
    if (a.nsp > 1) {
        const int n_cb = static_cast<int>((d_v + kMergeCols - 1) / kMergeCols);
        hipLaunchKernelGGL(attention_merge_kernel, dim3(static_cast<uint32_t>(a.n_hb * n_cb)), dim3(kAThreads),
                           a.merge_lds_bytes, s, p);
        if (hipGetLastError() != hipSuccess) return NMM_ERR_HIP;
    }
    return NMM_OK;
}

}  // extern "C"
