// The latent-attention workgroup (flash-decoding over a span of cache positions for a block of
// heads), shared by the attention launch and by the W_O launch that runs attention workgroups
// beside its GEMV workgroups.  The design is described where the attention launch is defined
// (attention.hip).
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
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kAWaves = 4;                // waves per attention workgroup, one per SIMD
constexpr int kAThreads = 64 * kAWaves;
constexpr int kCh = 64;                   // cache positions per chunk (16 per wave in Q.K^T)
constexpr int kMaxCols = 576;             // staged columns per cache row: max(d_qk, d_v)
constexpr int kPadSlots = 2;              // 16-byte padding slots after each staged row
constexpr int kPitchMax = kMaxCols + 8 * kPadSlots;   // 592 elements: LDS row pitch at 576 columns
constexpr int kMaxKs = kMaxCols / 32;     // Q.K^T k-steps (32 dims each)
constexpr int kMaxNtw = 8;                // P.V column tiles (16 columns) per wave: d_v <= 512
constexpr int kMaxHt = 2;                 // head tiles (16 heads) per workgroup, at most
constexpr int kHt = 2;                    // head tiles per workgroup beside a GEMV's
constexpr int kPPitch = kCh + 8;          // row pitch (elements) of P in LDS
constexpr int kKw = 6;                    // K fragments in flight in Q.K^T
constexpr int kRsrcWord3 = 0x00020000;
constexpr uint32_t kOutOfRange = 0x80000000u;
// A chunk rescales the running output only when its maximum exceeds the running reference by
// more than this (log2 units), so probabilities stay below 2^kLazyTh and the rescale is rare.
constexpr float kLazyTh = 8.f;

struct AttnParams {
    const uint16_t* q;
    int64_t ldq;
    const uint16_t* kv;
    int64_t ldkv;
    float* out;
    int64_t ldo;
    uint16_t* outb;     // optional bf16 copy of out (nearest, ties to even), outb[h * ldob + n]
    int64_t ldob;
    float* part_o;      // [n_hb][nsp][hb][d_v]: unnormalised span outputs (hb = heads per block)
    float* part_ml;     // [n_hb][nsp][hb][2]: the span's reference maximum and probability sum
    int heads, seq, dqk, dv;
    int cols;           // staged columns per cache row: max(d_qk, d_v)
    int pitch;          // LDS row pitch of a staged chunk (elements)
    int nsp, span, n_hb;
    int hbh;            // heads per block (16 per head tile)
    int xcd_map;        // 1: the head blocks of a span grouped on one XCD (grid padded to 8 spans)
    float scale_log2;   // scale * log2(e): scores are kept in log2 units
    uint32_t kv_extent; // bytes of the cache that may be read
    uint32_t q_extent;  // bytes of q that may be read
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kRsrcWord3);
}

__device__ __forceinline__ bf16x8 as_bf16x8(i32x4 v) { return __builtin_bit_cast(bf16x8, v); }

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

// Staging a chunk's cache rows into LDS: buffer loads that write LDS directly (no registers), one
// instruction moving 64 x 16 bytes into consecutive LDS slots, lane l into slot l.  A chunk is
// kCh rows of spr slots (cols / 8 data slots, then kPadSlots of padding), so instruction i covers
// slots 64 i .. 64 i + 63 and a chunk takes spr instructions; wave w of W issues i = w, w + W, ...
// stage_offsets computes once where each of this lane's slots lies in the cache relative to the
// chunk's first row (padding slots get an offset past any extent, so they read zeros); the chunk's
// row offset is added at issue.  Rows past the cache end fall outside the buffer's range and read
// zeros; a span's chunks never cross into the next span (spans are whole chunks).
template <int W>
struct Stage {
    static constexpr int kIns = (kPitchMax / 8 + W - 1) / W;   // instructions per wave
    static constexpr int kMinPieces = (kPitchMax / 8 - (W - 1) + W - 1) / W;   // the fewest any wave issues
    uint32_t off[kIns];
    __device__ __forceinline__ void init(int spr, int64_t ldkv, int wave, int lane) {
#pragma unroll
        for (int k = 0; k < kIns; ++k) {
            const int ins = wave + W * k;
            const int sl = ins * 64 + lane;
            const int row = sl / spr, c = sl - row * spr;
            off[k] = (ins < spr && c < spr - kPadSlots) ? uint32_t((int64_t(row) * ldkv + 8 * c) * 2) : kOutOfRange;
        }
    }
    __device__ __forceinline__ void piece(uint16_t* buf, __amdgpu_buffer_rsrc_t kvr, int k, int spr, uint32_t row_off,
                                          int wave) const {
        const int ins = wave + W * k;
        if (k < kIns && ins < spr)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(kvr, (lds_void*)(buf + ins * 64 * 8), 16, off[k] + row_off, 0, 0, 0);
    }
};

// A workgroup barrier for the LDS exchanges inside a chunk: this wave's LDS operations complete
// (lgkmcnt), then the barrier.  A fenced barrier (__syncthreads, or a fence on LDS alone) would
// also wait for the next chunk's staging loads, which write LDS through the vector memory counter,
// and so serialise the prefetch with the chunk; those loads target the other chunk buffer, which
// nothing reads before the end-of-chunk barrier waits for them.  The asm's memory clobber keeps
// the compiler from moving memory operations across it.
__device__ __forceinline__ void lds_sync() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Wait until at most N vector-memory operations of this wave are outstanding (N < 64).
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt holds 6 bits");
    // gfx9 encoding: vmcnt in bits 3:0 and 15:14; expcnt (6:4) and lgkmcnt (11:8) left at their maxima
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// LDS of the attention workgroup.  Every kernel that calls these gets the same arrays, so a kernel
// whose other workgroups do other work (the GEMV beside attention) can use them as well.
__device__ __forceinline__ uint16_t* chunk_buffer_a() {
    __shared__ __attribute__((aligned(16))) uint16_t kv_a[kCh * kPitchMax];
    return kv_a;
}
__device__ __forceinline__ uint16_t* chunk_buffer_b() {
    __shared__ __attribute__((aligned(16))) uint16_t kv_b[kCh * kPitchMax];
    return kv_b;
}
__device__ __forceinline__ uint16_t* p_buffer() {
    __shared__ __attribute__((aligned(16))) uint16_t pb[kMaxHt * 16 * kPPitch];
    return pb;
}
__device__ __forceinline__ float* red_buffer() {
    __shared__ __attribute__((aligned(16))) float red[4 * kMaxHt * 16];
    return red;
}
__device__ __forceinline__ int* flag_buffer() {
    __shared__ __attribute__((aligned(16))) int flags[8];
    return flags;
}

// The (head block x VS + column part, span) of workgroup `bid`, nb = n_hb x VS of the first; false
// for the padding workgroups of an XCD-grouped grid.  With xcd_map the workgroups of one span
// (every head block and column part) are 8 ids apart, so they run on one XCD and its L2 serves the
// span's cache rows to all of them.
__device__ __forceinline__ bool block_of(const AttnParams& p, int bid, int nb, int* hb, int* sp) {
    if (p.xcd_map) {
        *sp = (bid & 7) + 8 * (bid / (8 * nb));
        *hb = (bid >> 3) % nb;
        return *sp < p.nsp;
    }
    *hb = bid % nb;
    *sp = bid / nb;
    return true;
}

// One attention workgroup: HT * 16 heads (head block hb) over one span of positions, with 4 waves.
// Wave w is position group pw = w and covers all HT head tiles.  With VS = 2 or 4 that many
// workgroups share a (head block, span): all compute the scores and probabilities, and each the
// product with V, its stores and the merge's inputs for 1 / VS of d_v's column tiles (4 NTW tiles
// from tile0); the first also stores the reference and sum.  Each output column sees the same
// operations either way.
//  * Q.K^T: a wave computes the scores of positions 16 pw .. + 15 of each 64-position chunk for its
//    head tiles (S^T = K . Q^T on the matrix cores, K fragments read from LDS and used for each of
//    the wave's head tiles; Q held in registers as MFMA fragments).
//  * softmax: each wave writes P = 2^(s - reference), rounded to bf16, against the running
//    reference of each head, and posts its maxima.  Only when some wave's maximum exceeds a
//    reference by more than kLazyTh (always on a span's first chunk, rarely after) do the waves
//    take the chunk maximum, move the reference, rescale the output and write P again.  So
//    P <= 2^kLazyTh.
//  * P.V: a wave accumulates the output columns of tiles pw, pw + 4, ... for its head tiles
//    (O^T = V^T . P^T, V^T fragments by ds_read_b64_tr_b16 from the same staged rows).
//  * The result is stored straight from the accumulators, 64 contiguous bytes of 16 rows per store.
// KS = d_qk / 32 and NTW = column tiles per position group are upper bounds; EXACT: the shape
// matches them.
template <int HT, int KS, int NTW, bool EXACT, int VS = 1>
__device__ __forceinline__ void attention_block(const AttnParams p, int bid) {
    constexpr int W = kAWaves;
    constexpr int HB = 16 * HT;
    constexpr int HTW = HT;                    // head tiles per wave: all of them
    static_assert(W == 4 && HT >= 1 && HT <= kMaxHt, "one position group per wave, every wave over all head tiles");
    uint16_t* const kv_a = chunk_buffer_a();
    uint16_t* const kv_b = chunk_buffer_b();
    uint16_t* const pbuf = p_buffer();
    float* const red = red_buffer();
    int* const flags = flag_buffer();

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) & (W - 1);   // (the mask bounds it for the compiler)
    const int pw = wave;
    const int g = lane >> 4, j = lane & 15;
    const int ksteps = EXACT ? KS : p.dqk / 32;
    const int ntiles = EXACT ? 4 * NTW : p.dv / 16;
    const int pitch = EXACT ? kPitchMax : p.pitch;
    const int spr = pitch / 8;
    const uint32_t row_bytes = uint32_t(p.ldkv) * 2;

    static_assert(VS == 1 || VS == 2 || VS == 4, "one, two or four column parts");
    int hbv, sp;
    if (!block_of(p, bid, p.n_hb * VS, &hbv, &sp)) return;
    const int vh = hbv % VS, hb = hbv / VS;
    const int tile0 = vh * 4 * NTW;            // the workgroup's first 16-column tile of d_v
    const int h0 = hb * HB;
    const int s_begin = sp * p.span;
    const int s_end = min(p.seq, s_begin + p.span);
    const int nchunks = (s_end - s_begin + kCh - 1) / kCh;

    const __amdgpu_buffer_rsrc_t kvr = make_rsrc(p.kv, p.kv_extent);
    Stage<W> stg;
    stg.init(spr, p.ldkv, wave, lane);
    // ---- the block's Q rows to buffer b, then the first chunk to buffer a (LDS-direct loads of
    // whole row pieces: fragment-shaped global loads, 16 rows x 64 bytes per instruction, ingest
    // about four times slower).  Q rows past the last head and pieces past d_qk read zeros.  Q goes
    // first so that its fragments can be read while the chunk is still landing.
    {
        const __amdgpu_buffer_rsrc_t qr = make_rsrc(p.q, p.q_extent);
        const int qcols = ksteps * 4;                  // 16-byte pieces of a Q row that are read
        for (int ins = wave; ins * 64 < HB * spr; ins += W) {
            const int sl = ins * 64 + lane;
            const int row = sl / spr, c = sl - row * spr;
            const bool ok = c < qcols && h0 + row < p.heads;
            const uint32_t off = ok ? uint32_t((int64_t(h0 + row) * p.ldq + 8 * c) * 2) : kOutOfRange;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(qr, (lds_void*)(kv_b + ins * 64 * 8), 16, off, 0, 0, 0);
        }
    }
#pragma unroll
    for (int k = 0; k < Stage<W>::kIns; ++k) stg.piece(kv_a, kvr, k, spr, uint32_t(s_begin) * row_bytes, wave);
    // this wave's Q pieces have landed once at most its chunk pieces are outstanding (loads
    // complete in order; every wave issues at least kMinPieces of them at the full pitch), then
    // every wave's
    if constexpr (EXACT) wait_vm<Stage<W>::kMinPieces>();
    else __builtin_amdgcn_s_waitcnt(0);
    lds_sync();
    // the Q fragments of the wave's head tiles: head 16 t + j, dims 32 u + 8 g .. + 7; then
    // buffer b is free for chunk 1
    i32x4 qf[HTW][KS];
#pragma unroll
    for (int t = 0; t < HTW; ++t)
#pragma unroll
        for (int u = 0; u < KS; ++u)
            if (EXACT || u < ksteps)
                qf[t][u] = *reinterpret_cast<const i32x4*>(kv_b + (16 * t + j) * pitch + 8 * g + 32 * u);
    // the first chunk has landed: this wave's pieces, then every wave's
    __builtin_amdgcn_s_waitcnt(0);
    lds_sync();

    f32x4 o[NTW][HTW];      // O^T tiles: lane (g, j) holds columns 16 ct + 4 g .. + 3 of head 16 t + j
#pragma unroll
    for (int i = 0; i < NTW; ++i)
#pragma unroll
        for (int t = 0; t < HTW; ++t) o[i][t] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_ref[HTW], l_acc[HTW];   // the head's reference maximum (log2 units); this lane's sum of P
#pragma unroll
    for (int t = 0; t < HTW; ++t) {
        m_ref[t] = -INFINITY;
        l_acc[t] = 0.f;
    }
    const int a4 = j >> 2, b4 = j & 3;

    auto chunk = [&](const uint16_t* cur, uint16_t* nxt, int ck) {
        const int c0 = s_begin + ck * kCh;
        // the next chunk streams into the other buffer while this one is computed (every wave
        // finished reading that buffer before the last barrier); its loads are issued one per
        // Q.K^T step, so their issue overlaps the MFMAs instead of stalling the wave
        const bool stage_next = ck + 1 < nchunks;
        const uint32_t next_off = uint32_t(c0 + kCh) * row_bytes;

        // ---- S^T[16 positions][16 heads] per head tile; two accumulators per tile (even and odd
        // k-steps) keep two independent MFMA chains per tile in flight.  K fragments are read kKw
        // k-steps ahead: step u's MFMAs consume slot u % kKw, whose register then takes the read
        // of step u + kKw (kept next to them by a scheduling barrier), so LDS latency overlaps the
        // MFMAs instead of stalling every step.
        f32x4 s[HTW][2];
#pragma unroll
        for (int t = 0; t < HTW; ++t) s[t][0] = s[t][1] = f32x4{0.f, 0.f, 0.f, 0.f};
        const uint16_t* krow = cur + (16 * pw + j) * pitch + 8 * g;
        i32x4 kf[kKw];
#pragma unroll
        for (int u = 0; u < kKw; ++u)
            if (u < KS && (EXACT || u < ksteps)) kf[u] = *reinterpret_cast<const i32x4*>(krow + 32 * u);
#pragma unroll
        for (int u = 0; u < KS; ++u) {
            if (EXACT || u < ksteps) {
#pragma unroll
                for (int t = 0; t < HTW; ++t)
                    s[t][u & 1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kf[u % kKw]), as_bf16x8(qf[t][u]),
                                                                        s[t][u & 1], 0, 0, 0);
                if (u + kKw < KS && (EXACT || u + kKw < ksteps))
                    kf[u % kKw] = *reinterpret_cast<const i32x4*>(krow + 32 * (u + kKw));
                if (stage_next) stg.piece(nxt, kvr, u, spr, next_off, wave);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        // the staging pieces the Q.K^T steps did not issue
        if (stage_next) {
#pragma unroll
            for (int k = 0; k < Stage<W>::kIns; ++k)
                if (k >= KS || (!EXACT && k >= ksteps)) stg.piece(nxt, kvr, k, spr, next_off, wave);
        }

        // ---- scores in log2 units (positions past the span masked) and this wave's maximum per
        // head over its 16 positions
        const int pos0 = c0 + 16 * pw + 4 * g;
        float mx[HTW];
        bool need = false;
#pragma unroll
        for (int t = 0; t < HTW; ++t) {
            mx[t] = -INFINITY;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float v = (pos0 + i < s_end) ? (s[t][0][i] + s[t][1][i]) * p.scale_log2 : -INFINITY;
                s[t][0][i] = v;
                mx[t] = fmaxf(mx[t], v);
            }
            mx[t] = cols4_max(mx[t]);
            need |= !(mx[t] <= m_ref[t] + kLazyTh);
        }
        // ---- P = 2^(s - reference), rounded to bf16, to LDS as P[head][position]
        float lc[HTW];
        auto write_p = [&]() {
#pragma unroll
            for (int t = 0; t < HTW; ++t) {
                float pv[4];
                lc[t] = 0.f;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float v = s[t][0][i];
                    pv[i] = (v == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(v - m_ref[t]);
                    lc[t] += pv[i];
                }
                *reinterpret_cast<uint2*>(pbuf + (16 * t + j) * kPPitch + 16 * pw + 4 * g) =
                    uint2{pack_bf16(pv[0], pv[1]), pack_bf16(pv[2], pv[3])};
            }
        };
        // every wave posts its maxima and whether any moved past its reference by more than kLazyTh
        if (g == 0) {
#pragma unroll
            for (int t = 0; t < HTW; ++t) red[pw * HB + 16 * t + j] = mx[t];
        }
        if (ck > 0) {
            write_p();
            const bool wave_needs = __builtin_amdgcn_ballot_w64(need) != 0;
            if (lane == 0) flags[wave] = wave_needs ? 1 : 0;
            lds_sync();
        } else {
            lds_sync();   // a span's first chunk always sets the references
        }
        bool any = ck == 0;
        if (ck > 0) {
            // every wave's flag in one 16-byte LDS read
            const i32x4 f0 = *reinterpret_cast<const i32x4*>(flags);
            any = (f0[0] | f0[1] | f0[2] | f0[3]) != 0;
        }
        // ---- a reference moves (the same decision in every wave: all read the same maxima): the
        // chunk maximum of each head, the output rescaled, and P written again
        if (any) {
            bool resc = false;
            float alpha[HTW];
#pragma unroll
            for (int t = 0; t < HTW; ++t) {
                const int hh = 16 * t + j;
                const float mc = fmaxf(fmaxf(red[hh], red[HB + hh]), fmaxf(red[2 * HB + hh], red[3 * HB + hh]));
                alpha[t] = 1.f;
                if (mc > m_ref[t] + kLazyTh) {
                    alpha[t] = (m_ref[t] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_ref[t] - mc);
                    m_ref[t] = mc;
                    l_acc[t] *= alpha[t];
                    resc = true;
                }
            }
            if (__builtin_amdgcn_ballot_w64(resc)) {
#pragma unroll
                for (int i = 0; i < NTW; ++i)
#pragma unroll
                    for (int t = 0; t < HTW; ++t) o[i][t] *= alpha[t];
            }
            write_p();
            lds_sync();
        }
#pragma unroll
        for (int t = 0; t < HTW; ++t) l_acc[t] += lc[t];

        // ---- O^T += V^T . P^T over the chunk's two 32-position k-steps
#pragma unroll
        for (int kk = 0; kk < kCh / 32; ++kk) {
            i32x4 pf[HTW];
#pragma unroll
            for (int t = 0; t < HTW; ++t)
                pf[t] = *reinterpret_cast<const i32x4*>(pbuf + (16 * t + j) * kPPitch + 32 * kk + 8 * g);
            const uint16_t* vrow = cur + (32 * kk + 8 * g + a4) * pitch + 4 * b4;
            i32x4 vf[NTW];
#pragma unroll
            for (int i = 0; i < NTW; ++i) {
                const int ct = pw + 4 * i;
                if (EXACT || ct < ntiles) {
                    const uint16_t* base = vrow + 16 * (tile0 + ct);
                    const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(base));
                    const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(base + 4 * pitch));
                    const uint2 ulo = __builtin_bit_cast(uint2, lo), uhi = __builtin_bit_cast(uint2, hi);
                    vf[i] = i32x4{int(ulo.x), int(ulo.y), int(uhi.x), int(uhi.y)};
                }
            }
#pragma unroll
            for (int i = 0; i < NTW; ++i) {
                const int ct = pw + 4 * i;
                if (EXACT || ct < ntiles) {
#pragma unroll
                    for (int t = 0; t < HTW; ++t)
                        o[i][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vf[i]), as_bf16x8(pf[t]), o[i][t], 0, 0, 0);
                }
            }
        }

        // ---- the next chunk must have landed (this wave's loads, then every wave's), and every
        // wave must be done with this chunk's rows and P
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
    };
    for (int ck = 0; ck < nchunks; ck += 2) {
        chunk(kv_a, kv_b, ck);
        if (ck + 1 < nchunks) chunk(kv_b, kv_a, ck + 1);
    }

    // ---- the span's probability sums: this lane's positions, the wave's four rows, then the
    // four position groups in order
#pragma unroll
    for (int t = 0; t < HTW; ++t) {
        const float lw = cols4_sum(l_acc[t]);
        if (g == 0) red[pw * HB + 16 * t + j] = lw;
    }
    __syncthreads();
    float lsum[HTW];
#pragma unroll
    for (int t = 0; t < HTW; ++t) {
        const int hh = 16 * t + j;
        lsum[t] = ((red[hh] + red[HB + hh]) + red[2 * HB + hh]) + red[3 * HB + hh];
    }

    // ---- the block's [HB][d_v] result straight from the accumulators: lane (g, j) holds columns
    // 16 ct + 4 g .. + 3 of its head, so each store instruction writes 64 contiguous bytes of 16
    // rows; normalised when the span is the whole sequence, else the span's partial (stored
    // non-temporal: it is read once, by the merge on other XCDs)
    const bool whole = p.nsp == 1;
    const int64_t pidx = int64_t(hb) * p.nsp + sp;
#pragma unroll
    for (int t = 0; t < HTW; ++t) {
        const int row = 16 * t + j;
        const int h = h0 + row;
        if (whole) {
            if (h < p.heads) {
                const float scl = 1.f / lsum[t];
#pragma unroll
                for (int i = 0; i < NTW; ++i) {
                    const int ct = pw + 4 * i;
                    if (EXACT || ct < ntiles) {
                        const f32x4 v = o[i][t] * scl;
                        const int c = 16 * (tile0 + ct) + 4 * g;
                        *reinterpret_cast<f32x4*>(p.out + int64_t(h) * p.ldo + c) = v;
                        if (p.outb) {
                            uint16_t* d = p.outb + int64_t(h) * p.ldob + c;
                            d[0] = to_bf16_bits(v[0]);
                            d[1] = to_bf16_bits(v[1]);
                            d[2] = to_bf16_bits(v[2]);
                            d[3] = to_bf16_bits(v[3]);
                        }
                    }
                }
            }
        } else {
            float* const dst = p.part_o + (pidx * HB + row) * int64_t(p.dv) + 4 * g;
#pragma unroll
            for (int i = 0; i < NTW; ++i) {
                const int ct = pw + 4 * i;
                if (EXACT || ct < ntiles) __builtin_nontemporal_store(o[i][t], reinterpret_cast<f32x4*>(dst + 16 * (tile0 + ct)));
            }
            if (vh == 0 && pw == 0 && g == 0) *reinterpret_cast<float2*>(p.part_ml + (pidx * HB + row) * 2) = float2{m_ref[t], lsum[t]};
        }
    }
}

// Merge the spans of each head in span order:
//   out = sum_s w_s O_s / sum_s w_s l_s,  w_s = 2^(m_s - M),  M = max_s m_s.
// Lane s of every wave loads span s's (m, l) (at most 64 spans), so M and the normaliser come from
// one load and fixed-order butterflies; each thread loads its columns of every span at once and
// sums them in span order with explicit fused multiply-adds, the weights taken from lane s.  A
// block waits for about two memory round trips.  Two forms, which give the same bits (the same
// operations on every output, in the same order):
//  * merge_block: block `blk` owns one head and 256 of its columns, one per thread `tid` (heads x
//    ceil(d_v / 256) blocks of 256 threads): many light blocks, for the workgroups another
//    kernel's launch carries beside its own.
//  * merge_block_wide: a one-wave block `blk` owns 256 columns of one head (ceil(d_v / 256) blocks
//    per head, the same count as merge_block's), thread t taking four of them, so each load moves
//    1 KB of a span's row: the merge launch of the attention on its own.
constexpr int kMergeThreads = 256;
constexpr int kMergeBatch = 32;
constexpr int kMergeWideThreads = 64;    // threads per block of merge_block_wide (256 columns)
constexpr int kMergeWideBatch = 16;  // spans merge_block_wide loads at once

// M's weight of this lane's span and the normaliser sum_s w_s l_s, the same in every lane
__device__ __forceinline__ float2 merge_weights(const AttnParams& p, int64_t base, int lane) {
#pragma clang fp contract(off)
    float2 m_l = float2{-INFINITY, 0.f};
    if (lane < p.nsp) m_l = *reinterpret_cast<const float2*>(p.part_ml + (base + int64_t(lane) * p.hbh) * 2);
    float M = m_l.x;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) M = fmaxf(M, __shfl_xor(M, off));
    const float w = (m_l.x == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_l.x - M);
    float den = w * m_l.y;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) den += __shfl_xor(den, off);
    return float2{w, den};
}

__device__ __forceinline__ void merge_block(const AttnParams& p, int blk, int tid) {
    // no contraction of its own: every translation unit that inlines this rounds alike (the
    // products of the sum are explicit fused multiply-adds)
#pragma clang fp contract(off)
    const int n_cb = (p.dv + kMergeThreads - 1) / kMergeThreads;
    const int h = blk / n_cb, cb = blk - h * n_cb;
    const int n = cb * kMergeThreads + tid;
    const int lane = tid & 63;
    const int hb = h / p.hbh, hl = h - hb * p.hbh;
    const int64_t base = int64_t(hb) * p.nsp * p.hbh + hl;      // (block, span 0, head) row
    const float* src = p.part_o + base * p.dv + n;
    const int64_t o_step = int64_t(p.hbh) * p.dv;
    const bool active = n < p.dv;
    // the partial outputs first (their loads are independent of the weights)
    float v[kMergeBatch];
#pragma unroll
    for (int u = 0; u < kMergeBatch; ++u) v[u] = (active && u < p.nsp) ? src[u * o_step] : 0.f;
    const float2 wd = merge_weights(p, base, lane);
    float acc = 0.f;
    for (int s0 = 0; s0 < p.nsp; s0 += kMergeBatch) {
        if (s0 > 0) {
#pragma unroll
            for (int u = 0; u < kMergeBatch; ++u) v[u] = (active && s0 + u < p.nsp) ? src[(s0 + u) * o_step] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u)
            if (s0 + u < p.nsp) acc = __builtin_fmaf(__int_as_float(__builtin_amdgcn_readlane(__float_as_int(wd.x), s0 + u)), v[u], acc);
    }
    if (!active) return;
    const float r = acc / wd.y;
    p.out[int64_t(h) * p.ldo + n] = r;
    if (p.outb) p.outb[int64_t(h) * p.ldob + n] = to_bf16_bits(r);
}

__device__ __forceinline__ void merge_block_wide(const AttnParams& p, int blk) {
#pragma clang fp contract(off)
    const int tid = static_cast<int>(threadIdx.x);
    const int n_cb = (p.dv + 4 * kMergeWideThreads - 1) / (4 * kMergeWideThreads);
    const int h = blk / n_cb;
    const int c = (blk - h * n_cb) * 4 * kMergeWideThreads + 4 * tid;
    const int lane = tid & 63;
    const int hb = h / p.hbh, hl = h - hb * p.hbh;
    const int64_t base = int64_t(hb) * p.nsp * p.hbh + hl;
    const float* src = p.part_o + base * p.dv + c;
    const int64_t o_step = int64_t(p.hbh) * p.dv;
    const bool active = c < p.dv;
    f32x4 v[kMergeWideBatch];
#pragma unroll
    for (int u = 0; u < kMergeWideBatch; ++u)
        v[u] = (active && u < p.nsp) ? *reinterpret_cast<const f32x4*>(src + u * o_step) : f32x4{0.f, 0.f, 0.f, 0.f};
    const float2 wd = merge_weights(p, base, lane);
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < p.nsp; s0 += kMergeWideBatch) {
        if (s0 > 0) {
#pragma unroll
            for (int u = 0; u < kMergeWideBatch; ++u)
                v[u] = (active && s0 + u < p.nsp) ? *reinterpret_cast<const f32x4*>(src + (s0 + u) * o_step)
                                                  : f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int u = 0; u < kMergeWideBatch; ++u)
            if (s0 + u < p.nsp) {
                const float wu = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wd.x), s0 + u));
#pragma unroll
                for (int e = 0; e < 4; ++e) acc[e] = __builtin_fmaf(wu, v[u][e], acc[e]);
            }
    }
    if (!active) return;
    f32x4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = acc[e] / wd.y;
    *reinterpret_cast<f32x4*>(p.out + int64_t(h) * p.ldo + c) = r;
    if (p.outb) {
        uint16_t* d = p.outb + int64_t(h) * p.ldob + c;
#pragma unroll
        for (int e = 0; e < 4; ++e) d[e] = to_bf16_bits(r[e]);
    }
}

// A prepared attention call: kernel arguments, the attention grid (0: nothing to launch), the
// number of merge blocks (0: one span, no merge; merge_block and merge_block_wide take the same
// count) and the kernel variant.
constexpr int kAttnExact = 1;      // d_qk 576, d_v 512
constexpr int kAttnGeneral = 2;    // d_qk <= 576, d_v <= 512
struct AttnLaunch {
    AttnParams p{};
    int64_t grid = 0;
    int64_t merge_grid = 0;
    int variant = 0;
    int vsplit = 1;    // workgroups per (head block, span), each taking 1 / vsplit of d_v's columns (1, 2, 4)
};

}  // namespace attn

// The call prepared for workgroups that share a GEMV's launch: blocks of 32 heads (two head tiles),
// the spans of the attention launch of the same call, within the same workspace size.
nmm_status prepare_attention(const AttnArgs& a, void* workspace, size_t workspace_bytes, attn::AttnLaunch* out);
nmm_status launch_prepared_attention(const attn::AttnLaunch& l, hipStream_t s);   // attention, then merge
nmm_status launch_attention_merge(const attn::AttnLaunch& l, hipStream_t s);
nmm_status launch_attention_kernel(const attn::AttnLaunch& l, hipStream_t s);      // attention alone, no merge

}  // namespace nmm
