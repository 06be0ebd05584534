// The latent-attention workgroup (flash-decoding over a span of cache positions for 64 heads),
// shared by the attention launch and by the W_O launch that runs attention workgroups beside
// its GEMV workgroups.  The design is described where the attention launch is defined.
#pragma once

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "bf16_cast.h"
#include "nmm_internal.h"

namespace nmm {
namespace attn {

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
    int xcd_map;        // 1: spans grouped per XCD (grid of n_hb x nsp padded to a multiple of 8)
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

// One workgroup of the attention launch: workgroup `bid` of n_hb * nsp (head block, span).  CH
// positions per chunk, KS = d_qk / 32 k-steps and NT = d_v / 16 output tiles (upper bounds;
// EXACT: the shape matches them, so no step is skipped at run time), PMAX the largest row
// pitch (elements) the launch may use.  The two chunk buffers are separate LDS arrays and the
// chunk loop is unrolled by two, so that every LDS read names the buffer that is not being
// filled -- the compiler then need not wait for the filling loads before reading.
// The two chunk buffers of CH * PMAX elements (one LDS array each; every kernel that calls these
// gets the same two arrays, so a kernel whose workgroups do other work can use them as well).
template <int CH, int PMAX>
__device__ __forceinline__ uint16_t* chunk_buffer_a() {
    __shared__ __attribute__((aligned(16))) uint16_t kv_a[CH * PMAX];
    return kv_a;
}
template <int CH, int PMAX>
__device__ __forceinline__ uint16_t* chunk_buffer_b() {
    __shared__ __attribute__((aligned(16))) uint16_t kv_b[CH * PMAX];
    return kv_b;
}

template <int CH, int KS, int NT, int PMAX, bool EXACT>
__device__ __forceinline__ void attention_block(const AttnParams p, int bid) {
    uint16_t* const kv_a = chunk_buffer_a<CH, PMAX>();
    uint16_t* const kv_b = chunk_buffer_b<CH, PMAX>();
    constexpr int SPR = EXACT ? (KS * 32 > NT * 16 ? KS * 32 : NT * 16) / 8 + 1 : 0;   // LDS slots per row
    constexpr int CT = CH / 16;            // score tiles per chunk
    constexpr int PK = CH / 32;            // P.V k-steps per chunk

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, j = lane & 15;
    const int ksteps = EXACT ? KS : p.dqk / 32;
    const int ntiles = EXACT ? NT : p.dv / 16;

    int hb, sp;
    if (p.xcd_map) {
        sp = (bid & 7) + 8 * (bid / (8 * p.n_hb));
        hb = (bid >> 3) % p.n_hb;
        if (sp >= p.nsp) return;    // padding of the grid to whole groups of 8 spans
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

// A prepared attention call: kernel arguments, the attention grid (0: nothing to launch), the
// merge grid (0: one span, no merge) and the kernel variant.
constexpr int kAttnExact64 = 1;     // d_qk 576, d_v 512, 64-position chunks
constexpr int kAttnExact32 = 2;     // the same shape, 32-position chunks
constexpr int kAttnGeneral64 = 3;
constexpr int kAttnGeneral32 = 4;
struct AttnLaunch {
    AttnParams p{};
    int64_t grid = 0;
    int64_t merge_grid = 0;
    int variant = 0;
};

}  // namespace attn

nmm_status prepare_attention(const AttnArgs& a, void* workspace, size_t workspace_bytes, attn::AttnLaunch* out);
nmm_status launch_prepared_attention(const attn::AttnLaunch& l, hipStream_t s);   // attention, then merge
nmm_status launch_attention_merge(const attn::AttnLaunch& l, hipStream_t s);

}  // namespace nmm
