// Single-token latent attention on the matrix cores (gfx950), the decode step's independent
// dense work.  The paper's point is that narrow MatMuls moved off the matrix unit let
// independent matrix-unit work start earlier (Condition 1 "Data Independence", Section III-A;
// Section IV-A); this kernel is that independent work here, run on its own stream.
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
//    combines them in span order.  The spans of one head block sit on one XCD (workgroup ids 8
//    apart) so the cache rows they share are read from HBM once per XCD.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdlib>

#include "bf16_cast.h"
#include "nmm_internal.h"

namespace nmm {
namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr int kHB = 64;           // heads per workgroup (16 per wave)
constexpr int kAThreads = 256;
constexpr int kRsrcWord3 = 0x00020000;
constexpr uint32_t kOutOfRange = 0x80000000u;

struct AttnParams {
    const uint16_t* q;
    int64_t ldq;
    const uint16_t* kv;
    int64_t ldkv;
    float* out;
    int64_t ldo;
    uint16_t* outb;     // optional bf16 copy of out (nearest, ties to even), outb[h * ldob + n]
    int64_t ldob;
    float* part_o;      // [n_hb][nsp][64][d_v]
    float* part_ml;     // [n_hb][nsp][64][2]
    int heads, seq, dqk, dv;
    int cols;           // staged columns per cache row: max(d_qk, d_v)
    int pitch;          // LDS row pitch of a staged chunk (elements)
    int nsp, span, n_hb;
    int xcd_map;        // 1: spans grouped per XCD (nsp % 8 == 0)
    float scale_log2;   // scale * log2(e): scores are kept in log2 units
    uint32_t kv_extent; // bytes of the cache that may be read
    uint32_t q_extent;  // bytes of q that may be read
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kRsrcWord3);
}

__device__ __forceinline__ bf16x8 as_bf16x8(i32x4 v) { return __builtin_bit_cast(bf16x8, v); }

typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

// Row exchanges between the four 16-lane rows of a wave: permlane32_swap(a, b) gives
// ([a0 a1 b0 b1], [a2 a3 b2 b3]) and permlane16_swap(a, b) gives ([a0 b0 a2 b2], [a1 b1 a3 b3]),
// where a0..a3 are the rows of a.
__device__ __forceinline__ u32x2 swap32(unsigned a, unsigned b) { return __builtin_amdgcn_permlane32_swap(a, b, false, false); }
__device__ __forceinline__ u32x2 swap16(unsigned a, unsigned b) { return __builtin_amdgcn_permlane16_swap(a, b, false, false); }

// Every lane gets the max / sum of the four lanes of its column (a fixed order, so identical in
// all four and deterministic).
__device__ __forceinline__ float cols4_max(float x) {
    const u32x2 a = swap32(__float_as_uint(x), __float_as_uint(x));
    const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const u32x2 b = swap16(__float_as_uint(y), __float_as_uint(y));
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float cols4_sum(float x) {
    const u32x2 a = swap32(__float_as_uint(x), __float_as_uint(x));
    const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const u32x2 b = swap16(__float_as_uint(y), __float_as_uint(y));
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

__device__ __forceinline__ unsigned pack_bf16(float lo, float hi) {
    return unsigned(__builtin_bit_cast(uint16_t, static_cast<__bf16>(lo))) |
           (unsigned(__builtin_bit_cast(uint16_t, static_cast<__bf16>(hi))) << 16);
}

typedef __attribute__((address_space(3))) void lds_void;

// Stage a chunk's cache rows into LDS with buffer loads that write LDS directly (no registers):
// one instruction moves 64 x 16 bytes into consecutive LDS slots, lane l into slot l.  The
// chunk is viewed as CH rows of cpr + 1 slots (one slot of padding per row); slot s of the
// chunk holds piece (s / (cpr + 1), s % (cpr + 1)) of the rows c0 .. c0 + CH - 1, and padding
// slots and positions past the span read zeros.  Wave w issues instructions w, w + 4, ...
template <int CH, int SPR>
__device__ __forceinline__ void stage_chunk(uint16_t* buf, __amdgpu_buffer_rsrc_t kvr, const AttnParams& p, int c0,
                                            int s_end, int wave, int lane) {
    const int spr = SPR ? SPR : p.cols / 8 + 1;   // slots per row (a constant for the fixed shape)
    const int slots = CH * spr;
    for (int ins = wave; ins * 64 < slots; ins += 4) {
        const int sl = ins * 64 + lane;
        const int row = sl / spr, c = sl - row * spr;
        const bool ok = c < spr - 1 && c0 + row < s_end;
        const uint32_t off = ok ? uint32_t((int64_t(c0 + row) * p.ldkv + 8 * c) * 2) : kOutOfRange;
        if (sl < slots)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(kvr, (lds_void*)(buf + ins * 64 * 8), 16, off, 0, 0, 0);
    }
}

// CH positions per chunk, KS = d_qk / 32 k-steps and NT = d_v / 16 output tiles (upper bounds;
// EXACT: the shape matches them, so no step is skipped at run time), PMAX the largest row
// pitch (elements) the launch may use.  The two chunk buffers are separate LDS arrays and the
// chunk loop is unrolled by two, so that every LDS read names the buffer that is not being
// filled -- the compiler then need not wait for the filling loads before reading.
template <int CH, int KS, int NT, int PMAX, bool EXACT>
__global__ __launch_bounds__(kAThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void attention_kernel(const AttnParams p) {
    __shared__ __attribute__((aligned(16))) uint16_t kv_a[CH * PMAX];
    __shared__ __attribute__((aligned(16))) uint16_t kv_b[CH * PMAX];
    constexpr int SPR = EXACT ? (KS * 32 > NT * 16 ? KS * 32 : NT * 16) / 8 + 1 : 0;   // LDS slots per row
    constexpr int CT = CH / 16;            // score tiles per chunk
    constexpr int PK = CH / 32;            // P.V k-steps per chunk

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, j = lane & 15;
    const int ksteps = EXACT ? KS : p.dqk / 32;
    const int ntiles = EXACT ? NT : p.dv / 16;

    int hb, sp;
    const int bid = blockIdx.x;
    if (p.xcd_map) {
        sp = (bid & 7) + 8 * (bid / (8 * p.n_hb));
        hb = (bid >> 3) % p.n_hb;
    } else {
        hb = bid % p.n_hb;
        sp = bid / p.n_hb;
    }
    const int hw = hb * kHB + 16 * wave;   // this wave's first head
    const int s_begin = sp * p.span;
    const int s_end = min(p.seq, s_begin + p.span);
    const int nchunks = (s_end - s_begin + CH - 1) / CH;

    const __amdgpu_buffer_rsrc_t kvr = make_rsrc(p.kv, p.kv_extent);
    // ---- this wave's Q rows as A fragments (row j, dims 32u + 8g .. +7); heads past the end
    // read zeros.  Then the first chunk goes to LDS.
    i32x4 qf[KS];
    {
        const __amdgpu_buffer_rsrc_t qr = make_rsrc(p.q, p.q_extent);
        const bool ok = hw + j < p.heads;
        const uint32_t base = uint32_t((int64_t(hw + j) * p.ldq + 8 * g) * 2);
#pragma unroll
        for (int u = 0; u < KS; ++u)
            qf[u] = __builtin_amdgcn_raw_buffer_load_b128(qr, (ok && u < ksteps) ? base + 64 * u : kOutOfRange, 0, 0);
    }
    stage_chunk<CH, SPR>(kv_a, kvr, p, s_begin, s_end, wave, lane);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    f32x4 o[NT];                            // O^T tiles: lane (g, j) holds columns 16t + 4g + i of head j
#pragma unroll
    for (int t = 0; t < NT; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;   // this lane's head (column j), in log2 units
    const int a4 = j >> 2, b4 = j & 3;

    // one chunk: computed from `cur`; the next chunk streams into `nxt` meanwhile
    auto chunk = [&](const uint16_t* cur, uint16_t* nxt, int ck) {
        const int c0 = s_begin + ck * CH;

        // ---- S^T[CH positions][16 heads] = K . Q^T: lane (g, j) gets positions 16t + 4g + i of
        // head j.  The K fragments of step u + 1 are read while step u multiplies.
        f32x4 s[CT];
#pragma unroll
        for (int t = 0; t < CT; ++t) s[t] = f32x4{0.f, 0.f, 0.f, 0.f};
        const uint16_t* krow = cur + j * p.pitch + 8 * g;
        i32x4 kf[2][CT];
#pragma unroll
        for (int t = 0; t < CT; ++t) kf[0][t] = *reinterpret_cast<const i32x4*>(krow + 16 * t * p.pitch);
#pragma unroll
        for (int u = 0; u < KS; ++u) {
            if (EXACT || u < ksteps) {
                if (u + 1 < KS && (EXACT || u + 1 < ksteps)) {
#pragma unroll
                    for (int t = 0; t < CT; ++t)
                        kf[(u + 1) & 1][t] = *reinterpret_cast<const i32x4*>(krow + 16 * t * p.pitch + 32 * (u + 1));
                }
#pragma unroll
                for (int t = 0; t < CT; ++t)
                    s[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kf[u & 1][t]), as_bf16x8(qf[u]), s[t], 0, 0, 0);
            }
        }

        // the next chunk's rows stream into the other buffer during the softmax and P.V (every
        // wave finished reading that buffer before the last barrier)
        if (ck + 1 < nchunks) stage_chunk<CH, SPR>(nxt, kvr, p, c0 + CH, s_end, wave, lane);

        // ---- online softmax of head j over the chunk
        float mx = -INFINITY;
#pragma unroll
        for (int t = 0; t < CT; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                s[t][i] = (c0 + 16 * t + 4 * g + i < s_end) ? s[t][i] * p.scale_log2 : -INFINITY;
                mx = fmaxf(mx, s[t][i]);
            }
        const float m_new = fmaxf(m_run, cols4_max(mx));
        const float alpha = (m_run == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_run - m_new);
        float sum = 0.f;
#pragma unroll
        for (int t = 0; t < CT; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                s[t][i] = (s[t][i] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(s[t][i] - m_new);
                sum += s[t][i];
            }
        l_run = alpha * l_run + cols4_sum(sum);
        m_run = m_new;
#pragma unroll
        for (int t = 0; t < NT; ++t) o[t] *= alpha;

        // ---- O^T += V^T . P^T.  The B operand of k-step kk (positions 32kk + 8g + e of head j)
        // is tiles 2kk and 2kk + 1 of P, rounded to bf16 and moved between rows by two swaps;
        // tile t + 1's V^T fragment is read while tile t multiplies.
#pragma unroll
        for (int kk = 0; kk < PK; ++kk) {
            const f32x4 p0 = s[2 * kk], p1 = s[2 * kk + 1];
            const u32x2 x0 = swap32(pack_bf16(p0[0], p0[1]), pack_bf16(p1[0], p1[1]));
            const u32x2 x1 = swap32(pack_bf16(p0[2], p0[3]), pack_bf16(p1[2], p1[3]));
            const u32x2 y0 = swap16(x0[0], x0[1]);
            const u32x2 y1 = swap16(x1[0], x1[1]);
            const i32x4 pb = i32x4{int(y0[0]), int(y1[0]), int(y0[1]), int(y1[1])};
            const uint16_t* vrow = cur + (32 * kk + 8 * g + a4) * p.pitch + 4 * b4;
            auto vfrag = [&](int t) {
                const uint16_t* base = vrow + 16 * t;
                const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(base));
                const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(base + 4 * p.pitch));
                const uint2 ulo = __builtin_bit_cast(uint2, lo), uhi = __builtin_bit_cast(uint2, hi);
                return i32x4{int(ulo.x), int(ulo.y), int(uhi.x), int(uhi.y)};
            };
            i32x4 vb[2];
            vb[0] = vfrag(0);
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                if (EXACT || t < ntiles) {
                    if (t + 1 < NT && (EXACT || t + 1 < ntiles)) vb[(t + 1) & 1] = vfrag(t + 1);
                    o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vb[t & 1]), as_bf16x8(pb), o[t], 0, 0, 0);
                }
            }
        }

        // ---- the next chunk must have landed in LDS (this wave's loads, then every wave's)
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
    };
    for (int ck = 0; ck < nchunks; ck += 2) {
        chunk(kv_a, kv_b, ck);
        if (ck + 1 < nchunks) chunk(kv_b, kv_a, ck + 1);
    }

    // ---- this span's result: lane (g, j) holds columns 16t + 4g .. +3 of head hw + j
    const int h = hw + j;
    if (p.nsp == 1) {
        if (h < p.heads) {
            const float inv = 1.f / l_run;
#pragma unroll
            for (int t = 0; t < NT; ++t)
                if (EXACT || t < ntiles) {
                    const f32x4 r = o[t] * inv;
                    *reinterpret_cast<f32x4*>(p.out + int64_t(h) * p.ldo + 16 * t + 4 * g) = r;
                    if (p.outb) {
                        uint16_t* ob = p.outb + int64_t(h) * p.ldob + 16 * t + 4 * g;
                        ob[0] = to_bf16_bits(r[0]);
                        ob[1] = to_bf16_bits(r[1]);
                        ob[2] = to_bf16_bits(r[2]);
                        ob[3] = to_bf16_bits(r[3]);
                    }
                }
        }
        return;
    }
    const int64_t pidx = int64_t(hb) * p.nsp + sp;
    float* po = p.part_o + (pidx * kHB + 16 * wave + j) * int64_t(p.dv);
#pragma unroll
    for (int t = 0; t < NT; ++t)
        if (EXACT || t < ntiles) *reinterpret_cast<f32x4*>(po + 16 * t + 4 * g) = o[t];
    if (g == 0) {
        float* pml = p.part_ml + (pidx * kHB + 16 * wave + j) * 2;
        pml[0] = m_run;
        pml[1] = l_run;
    }
}

// Merge the spans of each head in span order:
//   out = sum_s w_s O_s,  w_s = 2^(m_s - M) / sum_q 2^(m_q - M) l_q,  M = max_s m_s.
// One output per thread: a workgroup owns 4 heads x 64 columns, so 64 threads read one
// 256-byte segment of a (head, span) row.  The partial outputs' loads go out first; the spans'
// (max, sum) pairs follow, one pair per thread, into LDS, where one thread per head forms the
// weights -- so the whole merge waits for about one memory round trip.
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
    if (tid < kMergeHeads) {
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
    a.xcd_map = (a.nsp % 8 == 0) ? 1 : 0;
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

nmm_status attention_common(int64_t heads, int64_t seq, int64_t d_qk, int64_t d_v, const void* q, int64_t ldq,
                            const void* kv, int64_t ld_kv, float scale, float* out, int64_t ldo, void* outb,
                            int64_t ldob, int64_t splits, void* workspace, size_t workspace_bytes, void* stream) {
    if (splits < 0) return NMM_ERR_ARG;
    AttnPlan a;
    nmm_status st = plan_attention(heads, seq, d_qk, d_v, &a, splits);
    if (st != NMM_OK) return st;
    if (!std::isfinite(scale)) return NMM_ERR_ARG;
    if (heads == 0) return NMM_OK;
    if (!q || !kv || !out) return NMM_ERR_NULL;
    if (ldq < d_qk || ld_kv < std::max(d_qk, d_v) || ldo < d_v) return NMM_ERR_SHAPE;
    if ((reinterpret_cast<uintptr_t>(q) & 15u) || (reinterpret_cast<uintptr_t>(kv) & 15u) || ldq % 8 ||
        ld_kv % 8 || (reinterpret_cast<uintptr_t>(out) & 15u) || ldo % 4)
        return NMM_ERR_ALIGN;
    const int64_t extent = ((seq - 1) * ld_kv + std::max(d_qk, d_v)) * 2;
    const int64_t q_extent = ((heads - 1) * ldq + d_qk) * 2;
    if (extent >= (int64_t(1) << 31) || q_extent >= (int64_t(1) << 31) || ldo >= (int64_t(1) << 31)) return NMM_ERR_SHAPE;
    st = validate_workspace(workspace, workspace_bytes, a.ws_bytes);
    if (st != NMM_OK) return st;

    AttnParams p{};
    p.q = static_cast<const uint16_t*>(q);
    p.ldq = ldq;
    p.kv = static_cast<const uint16_t*>(kv);
    p.ldkv = ld_kv;
    p.out = out;
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
    const int64_t grid = int64_t(a.n_hb) * a.nsp;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (d_qk == 576 && d_v == 512)
        st = a.ch == 64 ? launch_attention<64, 18, 32, 584, true>(p, grid, s)
                        : launch_attention<32, 18, 32, 584, true>(p, grid, s);
    else if (a.ch == 64)
        st = launch_attention<64, 18, 32, 584, false>(p, grid, s);
    else
        st = launch_attention<32, 32, 32, 1032, false>(p, grid, s);
    if (st != NMM_OK) return st;
    if (a.nsp > 1) {
        const int64_t merge_grid = ((heads + kMergeHeads - 1) / kMergeHeads) * ((d_v + kMergeCols - 1) / kMergeCols);
        hipLaunchKernelGGL(attention_merge_kernel, dim3(static_cast<uint32_t>(merge_grid)),
                           dim3(kAThreads), 0, s, p);
        if (hipGetLastError() != hipSuccess) return NMM_ERR_HIP;
    }
    return NMM_OK;
}

}  // namespace

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
