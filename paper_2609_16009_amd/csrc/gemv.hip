// Streaming narrow MatMul (GEMV) for gfx950: y[M,N] = x[M,K] . W[K,N], M <= 16 per launch.
//
// The paper's generalized vector MatMul (Algorithm 1, Section III-B) has three stages: each
// executor loads its blocks, multiplies and reduces them into partial sums stored in a global
// temporary buffer, then all executors wait for each other and a subset gathers the partial
// sums into C.  On MI355X the executors are 256-thread workgroups and the design is set by HBM:
//
//  * Init: a workgroup owns one K-slice of one column panel (plan.cpp).  It stages its slice of
//    x once into LDS as fp32 (the paper loads the token block once per executor, Algorithm 2).
//  * Compute: every lane streams 16-byte chunks (8 columns of one row) of W with buffer loads
//    marked non-temporal, keeping U row-steps in flight, widens them exactly to fp32 (bf16: a
//    16-bit shift; fp16: the mixed-precision FMA) and accumulates x[m,k] * W[k,n] in fp32
//    registers.  W is read exactly once.
//  * Gather: the workgroup reduces its waves' partial sums through LDS in a fixed order.  If the
//    panel has one K-slice it writes y directly; otherwise it stores its partial sums to the
//    workspace, releases them at device scope and takes a ticket; the last workgroup of the
//    panel acquires and sums the slices in order 0..ks-1 (the paper's WaitAllVectors + Acc
//    loop, without a second launch), writes y and resets the ticket.  The order never depends
//    on which workgroup arrives last, so results are bit-reproducible.
//  * Optionally the gather also writes y rounded to bf16 (ties to even, the hardware
//    conversion) into a sliced layout: Algorithm 2's output cast, used to hand the next MatMul
//    of the decode chain its 16-bit operand without an extra kernel.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdlib>

#include "attention_core.h"
#include "bf16_cast.h"
#include "handoff.h"
#include "nmm_internal.h"

namespace nmm {
namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

// Buffer-resource word 3 for raw (unswizzled) gfx9 buffers; out-of-range reads return zero.
constexpr int kRsrcWord3 = 0x00020000;
// Cache policy of the W stream: non-temporal (read once, do not keep in the caches).
constexpr int kLoadNT = 2;

struct KParams {
    const uint16_t* x;
    int64_t ldx, sx;
    const uint16_t* w;
    int64_t sw;
    float* y;
    int64_t ldy, sy;
    uint16_t* ybf;
    int64_t ybf_group, ybf_keep, ybf_ldm, ybf_sb;
    int ybf_away;          // bf16 rounding of ybf: 0 nearest-even, 1 nearest with ties away from zero
    float* part;
    unsigned* tickets;
    int M, K, N;
    uint32_t row_bytes;   // ldw * 2
    uint32_t w_extent;    // bytes of one W: (K-1)*ldw*2 + roundup(N,8)*2
    int n_full, full_lg, tail_chunks, tail_lg;
    int ks_full, rows_full, ks_tail, rows_tail, ks_max;
    int items, mblocks, n_panels;
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kRsrcWord3);
}

template <int DT>
__device__ __forceinline__ float widen1(uint16_t h) {
    if constexpr (DT == NMM_BF16) {
        return __uint_as_float(uint32_t(h) << 16);
    } else {
        return static_cast<float>(__builtin_bit_cast(_Float16, h));
    }
}

// acc[m][j] += x[m] * W[j] for the 8 columns of one chunk.
template <int DT, int MT>
__device__ __forceinline__ void fma_chunk(float (&acc)[MT][8], const i32x4 v, const float* __restrict__ xr) {
    float xv[MT];
    if constexpr (MT >= 4) {
#pragma unroll
        for (int q = 0; q < MT / 4; ++q) {
            const f32x4 t = *reinterpret_cast<const f32x4*>(xr + 4 * q);
            xv[4 * q + 0] = t[0];
            xv[4 * q + 1] = t[1];
            xv[4 * q + 2] = t[2];
            xv[4 * q + 3] = t[3];
        }
    } else {
#pragma unroll
        for (int m = 0; m < MT; ++m) xv[m] = xr[m];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t u = static_cast<uint32_t>(v[i]);
        float lo, hi;
        if constexpr (DT == NMM_BF16) {
            lo = __uint_as_float(u << 16);
            hi = __uint_as_float(u & 0xFFFF0000u);
        } else {
            const f16x2 h = __builtin_bit_cast(f16x2, u);
            lo = static_cast<float>(h[0]);
            hi = static_cast<float>(h[1]);
        }
#pragma unroll
        for (int m = 0; m < MT; ++m) {
            acc[m][2 * i] = __builtin_fmaf(xv[m], lo, acc[m][2 * i]);
            acc[m][2 * i + 1] = __builtin_fmaf(xv[m], hi, acc[m][2 * i + 1]);
        }
    }
}

// An offset no W extent reaches (extents are < 2^31 bytes): a raw buffer load there returns 0.
constexpr uint32_t kOutOfRange = 0x80000000u;

// One 16-byte chunk of W.  In the guarded (last) K-slice, rows at or past K read as zeros
// through the buffer's range check instead of a branch, so the load stream stays straight-line.
template <bool GUARD>
__device__ __forceinline__ i32x4 load_chunk(__amdgpu_buffer_rsrc_t rsrc, uint32_t off, bool in_range) {
    if constexpr (GUARD) off = in_range ? off : kOutOfRange;
    return __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, kLoadNT);
}

// Where one lane reads W: a 16-byte column chunk, one row every `rstep` rows.
struct Stream {
    __amdgpu_buffer_rsrc_t rsrc;
    uint32_t off;         // byte offset of the lane's first chunk
    uint32_t step_bytes;  // rstep rows
    int row;              // the lane's first row
    int rstep;
    int K;
};

template <int U, bool GUARD>
__device__ __forceinline__ void prefetch(i32x4 (&buf)[U], const Stream& st) {
#pragma unroll
    for (int u = 0; u < U; ++u)
        buf[u] = load_chunk<GUARD>(st.rsrc, st.off + u * st.step_bytes, st.row + u * st.rstep < st.K);
}

// Consume `nsteps` row-steps (a multiple of U, the first U already in `buf`), keeping U loads in
// flight: step s is multiplied and its register then takes the load for step s+U.  Consuming a
// slot before reloading it lets every slot stay in one register across iterations (a load into
// a fresh register would have to be copied back at the end of the iteration, which waits for
// it), and a scheduling barrier keeps each reload next to its multiply.  The steady-state loop
// has no branches, so the wait counters track each load.
template <int DT, int MT, int U, bool GUARD>
__device__ __forceinline__ void stream_rows(float (&acc)[MT][8], i32x4 (&buf)[U], const Stream& st,
                                            int nsteps, const float* __restrict__ xs, int xs_step) {
    int s = 0;
    for (; s + U < nsteps; s += U) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            fma_chunk<DT, MT>(acc, buf[u], xs + (s + u) * xs_step);
            const int sn = s + U + u;
            buf[u] = load_chunk<GUARD>(st.rsrc, st.off + sn * st.step_bytes, st.row + sn * st.rstep < st.K);
            // keep the reload here: sunk to the end of the iteration it would leave nothing in
            // flight while the other slots are multiplied
            __builtin_amdgcn_sched_barrier(0);
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) fma_chunk<DT, MT>(acc, buf[u], xs + (s + u) * xs_step);
}

// How y and its bf16 copy are stored.  After MatMul 2 the fp32 y is read by the launch's last
// workgroup (the cache-entry epilogue), so there y goes out as device-scope atomic stores
// (coherent at memory).
constexpr int kStorePlain = 0;   // plain stores
constexpr int kStoreEpi = 2;     // y coherent
constexpr int kStoreNoY = 3;     // separate launch with the bf16 copy only (y is null)

// y[m, n] (fp32) and its optional bf16 copy.
template <int SM>
__device__ __forceinline__ void store_out(const KParams& p, int64_t b, int m, int n, float v) {
    if constexpr (SM != kStoreNoY) {
        float* yd = p.y + b * p.sy + int64_t(m) * p.ldy + n;
        if constexpr (SM == kStoreEpi) __hip_atomic_store(yd, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        else *yd = v;
    }
    if (p.ybf) {
        const int64_t g = n / p.ybf_group, r = n - g * p.ybf_group;
        if (r < p.ybf_keep) {
            uint16_t* dst = p.ybf + b * p.ybf_sb + int64_t(m) * p.ybf_ldm + g * p.ybf_keep + r;
            *dst = to_bf16_mode(v, p.ybf_away);
        }
    }
}

// Stage x[m0:m0+MT, k0:k0+rows] into LDS as fp32, layout [row][m], zero outside M x K, in two
// halves: stage_x_issue issues every 16-byte chunk load of the slice (8 consecutive k of one x
// row; chunks past x's extent read as zeros) and stage_x_commit widens them into LDS.  W loads
// issued between the two stay in flight while x is committed (loads complete in issue order).
constexpr int kXPer = (kXStageBytes / 4 / 8 + kThreads - 1) / kThreads;   // x chunks per thread

template <int MT, int AUX>
__device__ __forceinline__ void stage_x_issue(i32x4 (&v)[kXPer], const KParams& p, int64_t b, int m0, int k0,
                                              int rows, int tid) {
    const int cpr = rows / 8;                       // chunks per x row of the slice
    const int total = cpr * MT;
    const int mrows = min(MT, p.M - m0);
    // the row block's x: its extent reaches the 16-byte chunk holding each row's last element
    // (ABI rule; below 2 GiB by validation)
    const uint32_t x_extent = uint32_t((int64_t(mrows - 1) * p.ldx + (p.K + 7) / 8 * 8) * 2);
    const __amdgpu_buffer_rsrc_t xr = make_rsrc(p.x + b * p.sx + int64_t(m0) * p.ldx, x_extent);
#pragma unroll
    for (int j = 0; j < kXPer; ++j) {
        const int i = tid + j * kThreads;
        const int m = i / cpr, q = i - m * cpr;
        const bool ok = i < total && m < mrows;
        const uint32_t off = ok ? uint32_t((int64_t(m) * p.ldx + k0 + 8 * q) * 2) : kOutOfRange;
        v[j] = __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, AUX);
    }
}

template <int DT, int MT>
__device__ __forceinline__ void stage_x_commit(float* __restrict__ lds, const i32x4 (&v)[kXPer], const KParams& p,
                                               int k0, int rows, int tid) {
    const int cpr = rows / 8;
    const int total = cpr * MT;
#pragma unroll
    for (int j = 0; j < kXPer; ++j) {
        const int i = tid + j * kThreads;
        if (i < total) {
            const int m = i / cpr, q = i - m * cpr;
            const int kb = k0 + 8 * q;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const uint16_t h = static_cast<uint16_t>(uint32_t(v[j][e >> 1]) >> (16 * (e & 1)));
                lds[(8 * q + e) * MT + m] = (kb + e < p.K) ? widen1<DT>(h) : 0.f;
            }
        }
    }
}

// ---------------------------------------------------------------------------------------------
// One work item: one K-slice of one panel of one (batch entry, row block).
// ---------------------------------------------------------------------------------------------
struct Item {
    int64_t b;                    // batch entry
    int mb;                       // row block
    int panel, slice, ks, rows, valid;
    int lg, cw, c, rstep, rin;
    int k0, m0, chunk0;
};

template <int MT>
__device__ __forceinline__ Item item_of(const KParams& p, uint32_t bid, int tid) {
    Item it;
    const int lane = tid & 63, wave = tid >> 6;
    const int item = static_cast<int>(bid % uint32_t(p.items));
    const uint32_t bm = bid / uint32_t(p.items);
    it.mb = static_cast<int>(bm % uint32_t(p.mblocks));
    it.b = bm / uint32_t(p.mblocks);
    if (item < p.n_full * p.ks_full) {
        it.panel = item / p.ks_full;
        it.slice = item - it.panel * p.ks_full;
        it.lg = p.full_lg;
        it.ks = p.ks_full;
        it.rows = p.rows_full;
        it.valid = 1 << p.full_lg;
    } else {
        it.panel = p.n_full;
        it.slice = item - p.n_full * p.ks_full;
        it.lg = p.tail_lg;
        it.ks = p.ks_tail;
        it.rows = p.rows_tail;
        it.valid = p.tail_chunks;
    }
    it.cw = 1 << it.lg;                        // lanes across the panel's columns
    it.c = lane & (it.cw - 1);
    it.rstep = kWaves << (6 - it.lg);          // rows per workgroup step
    it.rin = wave * (64 >> it.lg) + (lane >> it.lg);
    it.k0 = it.slice * it.rows;
    it.m0 = it.mb * MT;
    it.chunk0 = it.panel << p.full_lg;         // first 8-column chunk of the panel
    return it;
}

// Where the item's lane reads W; lanes past a ragged panel edge re-read its last chunk.
__device__ __forceinline__ Stream stream_of(const KParams& p, const Item& it) {
    Stream st;
    const int cc = it.c < it.valid ? it.c : it.valid - 1;
    st.rsrc = make_rsrc(p.w + it.b * p.sw, p.w_extent);
    st.off = uint32_t(it.k0 + it.rin) * p.row_bytes + uint32_t(it.chunk0 + cc) * 16u;
    st.step_bytes = uint32_t(it.rstep) * p.row_bytes;
    st.row = it.k0 + it.rin;
    st.rstep = it.rstep;
    st.K = p.K;
    return st;
}

template <int MT>
__device__ __forceinline__ int64_t part_base(const KParams& p, const Item& it) {
    return (((it.b * p.mblocks + it.mb) * p.n_panels + it.panel) * int64_t(p.ks_max)) * (int64_t(MT) * kPanelCols);
}

// A workgroup barrier that orders LDS only.  __syncthreads() also releases global memory, which
// makes every wave wait for its outstanding stores first.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Row-group butterfly without LDS.  Within each 16-lane row, DPP rotations by 1, 2, 4 and 8 add
// lane l - off (mod 16) to lane l; applied for off = cw, 2cw, .. 8 they leave in every lane the sum
// of the row's lanes congruent to it mod cw (for off = 8 the partner is lane l ^ 8).  Across rows,
// v_permlane16_swap and v_permlane32_swap exchange 16-lane rows (permlane16_swap(x, x) gives the
// rows [x0 x0 x2 x2] and [x1 x1 x3 x3], permlane32_swap(x, x) gives [x0 x1 x0 x1] and
// [x2 x3 x2 x3], so the two halves add up to the pair sums x[l] + x[l ^ 16], x[l] + x[l ^ 32]).
template <int OFF>
__device__ __forceinline__ float add_ror(float x) {
    return x + __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x120 + OFF /* row_ror:OFF */, 0xF, 0xF, false));
}
__device__ __forceinline__ float add_xor16(float x) {
    const u32x2 r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r.x) + __uint_as_float(r.y);
}
__device__ __forceinline__ float add_xor32(float x) {
    const u32x2 r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r.x) + __uint_as_float(r.y);
}

// Gather, part 1: each wave folds its row groups with the butterfly above (lanes r*cw + c and
// r'*cw + c hold the same columns), then the four waves are summed through LDS in wave order.  A panel with one K-slice writes y; otherwise the slice's partial
// sums go to the workspace with device-scope stores (coherent past the per-XCD L2 caches).
template <int MT, int SM>
__device__ __forceinline__ void reduce_item(const KParams& p, const Item& it, float (&acc)[MT][8], float* lds,
                                            int tid) {
    const int lane = tid & 63, wave = tid >> 6;
#define NMM_FOLD(COND, OP)                                                   \
    if (COND) {                                                              \
        _Pragma("unroll") for (int m = 0; m < MT; ++m)                       \
            _Pragma("unroll") for (int j = 0; j < 8; ++j) acc[m][j] = OP(acc[m][j]); \
    }
    NMM_FOLD(it.cw <= 1, add_ror<1>)   // narrow tail panels only
    NMM_FOLD(it.cw <= 2, add_ror<2>)
    NMM_FOLD(it.cw <= 4, add_ror<4>)
    NMM_FOLD(it.cw <= 8, add_ror<8>)
    NMM_FOLD(it.cw <= 16, add_xor16)
    NMM_FOLD(it.cw <= 32, add_xor32)
#undef NMM_FOLD
    constexpr int MG = MT < 4 ? MT : 4;
    const int pcols = it.cw * 8;
    const int64_t pbase = part_base<MT>(p, it);
#pragma unroll
    for (int g = 0; g < MT; g += MG) {
        if (lane < it.cw) {
#pragma unroll
            for (int mm = 0; mm < MG; ++mm) {
                float* dst = lds + ((wave * MG + mm) * it.cw + it.c) * 8;
                *reinterpret_cast<f32x4*>(dst) = f32x4{acc[g + mm][0], acc[g + mm][1], acc[g + mm][2], acc[g + mm][3]};
                *reinterpret_cast<f32x4*>(dst + 4) = f32x4{acc[g + mm][4], acc[g + mm][5], acc[g + mm][6], acc[g + mm][7]};
            }
        }
        lds_barrier();
        for (int o = tid; o < MG * pcols; o += kThreads) {
            const int mm = o / pcols, col = o - mm * pcols;
            float v = lds[mm * pcols + col];
#pragma unroll
            for (int w = 1; w < kWaves; ++w) v += lds[(w * MG + mm) * pcols + col];
            const int m = g + mm;
            const int n = it.chunk0 * 8 + col;
            if (it.ks == 1) {
                if (it.m0 + m < p.M && n < p.N) store_out<SM>(p, it.b, it.m0 + m, n, v);
            } else {
                __hip_atomic_store(p.part + pbase + int64_t(it.slice) * (MT * kPanelCols) + m * kPanelCols + col,
                                   v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        lds_barrier();
    }
}

// Gather, part 2 (the panel's last workgroup only): every output of the panel sums its K-slices
// in slice order; the loads of R outputs x QB slices are all in flight before any is added.
template <int MT, int SM>
__device__ __forceinline__ void gather_panel(const KParams& p, const Item& it, int tid) {
    constexpr int R = (MT * 2 < 8) ? MT * 2 : 8;   // outputs per thread per pass (pcols <= 512)
    constexpr int QB = 32 / R;                      // slices per batch
    const int pcols = it.cw * 8;
    const int n_out = MT * pcols;
    const int64_t pbase = part_base<MT>(p, it);
    for (int o0 = tid; o0 < n_out; o0 += R * kThreads) {
        float sum[R];
#pragma unroll
        for (int r = 0; r < R; ++r) sum[r] = 0.f;
        for (int q0 = 0; q0 < it.ks; q0 += QB) {
            float v[R][QB];
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int o = o0 + r * kThreads;
                const int m = o / pcols, col = o - m * pcols;
                const float* src = p.part + pbase + m * kPanelCols + col;
#pragma unroll
                for (int u = 0; u < QB; ++u)
                    v[r][u] = (o < n_out && q0 + u < it.ks)
                                  ? __hip_atomic_load(src + int64_t(q0 + u) * (MT * kPanelCols), __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT)
                                  : 0.f;
            }
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int u = 0; u < QB; ++u)
                    if (q0 + u < it.ks) sum[r] += v[r][u];
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int o = o0 + r * kThreads;
            const int m = o / pcols, col = o - m * pcols;
            const int n = it.chunk0 * 8 + col;
            if (o < n_out && it.m0 + m < p.M && n < p.N) store_out<SM>(p, it.b, it.m0 + m, n, sum[r]);
        }
    }
}

// The panel's arrival counter (see arrive()).
__device__ __forceinline__ unsigned* ticket_of(const KParams& p, const Item& it) {
    return p.tickets + (it.b * p.mblocks + it.mb) * p.n_panels + it.panel;
}

// A work item's stream: stage its x slice, then multiply its K-slice of the panel into acc.
template <int DT, int MT, int U>
__device__ __forceinline__ void stream_item(const KParams& p, const Item& it, float* lds, float (&acc)[MT][8],
                                            int tid) {
    // ---- init: issue x's loads, then the first U loads of W, then commit x to LDS while the W
    // loads are still in flight
    const Stream st = stream_of(p, it);
    i32x4 xv[kXPer];
    stage_x_issue<MT, 0>(xv, p, it.b, it.m0, it.k0, it.rows, tid);
    i32x4 buf[U];
    prefetch<U, true>(buf, st);   // one straight-line path, so x's wait leaves these in flight
    stage_x_commit<DT, MT>(lds, xv, p, it.k0, it.rows, tid);
    __syncthreads();

    // ---- compute: stream this workgroup's rows of the panel
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[m][j] = 0.f;
    {
        const int nsteps = it.rows / it.rstep;
        const float* xs = lds + it.rin * MT;
        stream_rows<DT, MT, U, true>(acc, buf, st, nsteps, xs, it.rstep * MT);
    }
    __syncthreads();   // x slice no longer needed: LDS becomes the reduction buffer
}

// The gather of one panel (reduce_item has run): a single K-slice has written y already;
// otherwise the slice takes the panel's ticket and the last to arrive sums the slices.  Returns
// whether this workgroup wrote the panel's final outputs.
template <int MT, int SM>
__device__ __forceinline__ bool finish_panel(const KParams& p, const Item& it, int* s_last, int tid) {
    if (it.ks == 1) return true;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) {
        *s_last = arrive(ticket_of(p, it), unsigned(it.ks));
    }
    __syncthreads();
    if (!*s_last) return false;
    gather_panel<MT, SM>(p, it, tid);
    return true;
}

// One work item of a separate GEMV launch (SM: kStorePlain or kStoreNoY).
template <int DT, int MT, int U, int SM>
__device__ __forceinline__ void gemv_item(const KParams& p, uint32_t bid, float* lds, int* s_last) {
    const int tid = threadIdx.x;
    const Item it = item_of<MT>(p, bid, tid);
    float acc[MT][8];
    stream_item<DT, MT, U>(p, it, lds, acc, tid);
    reduce_item<MT, SM>(p, it, acc, lds, tid);
    (void)finish_panel<MT, SM>(p, it, s_last, tid);
}

template <int DT, int MT, int U, int SM>
__global__ __launch_bounds__(kThreads) void gemv_kernel(const KParams p) {
    extern __shared__ float lds[];
    __shared__ int s_last;
    gemv_item<DT, MT, U, SM>(p, blockIdx.x, lds, &s_last);
}

// A bf16 single-row GEMV and an independent latent attention in one launch: workgroups
// [0, attn_grid) are attention's, each a workgroup of the attention launch (dispatched first, so
// they start as early as the GEMV's), the rest are the GEMV's, exactly as in its own launch (item
// id = workgroup id - attn_grid, a multiple of 8, so every item keeps its XCD), the x slice
// staged in the first of attention's two chunk buffers.  The paper overlaps narrow MatMuls with independent matrix-core work (Condition 1 of
// Section III-A); here the overlap is fixed by the launch itself -- the GEMV's workgroups stream
// the weight while attention's run on the compute units the GEMV leaves free -- instead of
// depending on how two streams are scheduled.
static_assert(kThreads == attn::kAThreads, "the two kinds of workgroup have the same size");
static_assert(size_t(attn::kCh) * attn::kPitchMax * 2 >= size_t(kXStageBytes) && size_t(attn::kCh) * attn::kPitchMax * 2 >= size_t(kRedBytes),
              "the GEMV's x slice and reduction fit the first chunk buffer");
template <int U>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void gemv_attention_kernel(const KParams p, const attn::AttnParams a, uint32_t attn_grid) {
    __shared__ int s_last;
    if (blockIdx.x < attn_grid) {
        attn::attention_block<attn::kHt, attn::kMaxKs, attn::kMaxNtw, true>(a, static_cast<int>(blockIdx.x));
    } else {
        float* lds = reinterpret_cast<float*>(attn::chunk_buffer_a());
        gemv_item<NMM_BF16, 1, U, kStorePlain>(p, blockIdx.x - attn_grid, lds, &s_last);
    }
}

// A bf16 single-row GEMV with the merge of an attention launched earlier beside it: workgroups
// [0, gemv_grid) are the GEMV's (exactly as in its own launch), the rest take the merge's blocks
// in turn.  The merge reads only the attention's span partials, so it runs under the GEMV's
// weight stream instead of after it.
template <int U>
__global__ __launch_bounds__(kThreads) void gemv_merge_kernel(const KParams p, const attn::AttnParams a,
                                                             uint32_t gemv_grid, uint32_t merge_blocks) {
    extern __shared__ float lds[];
    __shared__ int s_last;
    if (blockIdx.x < gemv_grid) {
        gemv_item<NMM_BF16, 1, U, kStorePlain>(p, blockIdx.x, lds, &s_last);
    } else {
        const uint32_t n = gridDim.x - gemv_grid;
        for (uint32_t b = blockIdx.x - gemv_grid; b < merge_blocks; b += n)
            attn::merge_block(a, static_cast<int>(b), static_cast<int>(threadIdx.x));
    }
}

// ---------------------------------------------------------------------------------------------
// The transposed-weight GEMV: y[m, n] = sum_k x[m, k] * Wt[n, k] for Wt row-major [N, K] (the
// layout of a torch Linear weight, and the one a dense y = x Wt^T GEMM reads).  Each output is
// the dot product of two contiguous rows, so one load of a wave covers 512 k of one Wt row
// (64 lanes x 16 bytes), U loads stay in flight across the wave's rows, and each row is finished
// by the cross-lane butterfly once its last chunk is in: no cross-wave reduction.  A workgroup
// owns 4 r consecutive rows (r per wave) of one K-slice; K is split only where x's slice would
// not fit the LDS staging buffer, and then combined like the GEMV's panels (device-scope
// partials, one ticket per row block, the last arriver sums the slices in order).
// ---------------------------------------------------------------------------------------------
struct NtParams {
    const uint16_t* x;
    int64_t ldx;
    const uint16_t* wt;
    uint32_t row_bytes;      // ldwt * 2
    uint32_t w_extent;       // bytes of Wt: (N-1)*ldwt*2 + roundup(K, 8)*2
    float* y;
    int64_t ldy;
    float* part;
    unsigned* tickets;
    int M, K, N;
    int r;                   // rows per wave
    int slice_k;             // k per K-slice (a multiple of 512)
    int ks, row_blocks, mblocks;
};

constexpr int kNtChunk = 512;     // k covered by one wave-load
constexpr int kNtXPer = kXStageBytes / 16 / kThreads;   // 16-byte x chunks staged per thread

// x[m0 : m0+MT, k0 : k0+span] into LDS as raw 16-bit values, layout [k][m], zero past M and K
// (span a multiple of 8, span * MT * 2 <= kXStageBytes): the loads, then the LDS stores.
template <int MT>
__device__ __forceinline__ void nt_stage_x_issue(i32x4 (&v)[kNtXPer], const NtParams& p, int m0, int k0, int span,
                                                 int tid) {
    const int cpr = span / 8;
    const int mrows = min(MT, p.M - m0);
    const uint32_t x_extent = uint32_t((int64_t(mrows - 1) * p.ldx + (p.K + 7) / 8 * 8) * 2);
    const __amdgpu_buffer_rsrc_t xr = make_rsrc(p.x + int64_t(m0) * p.ldx, x_extent);
#pragma unroll
    for (int c = 0; c < kNtXPer; ++c) {
        const int i = tid + c * kThreads;
        const int m = i / cpr, q = i - m * cpr;
        const bool ok = i < cpr * MT && m < mrows && k0 + 8 * q < p.K;
        const uint32_t off = ok ? uint32_t((int64_t(m) * p.ldx + k0 + 8 * q) * 2) : kOutOfRange;
        v[c] = __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0);
    }
}

template <int MT>
__device__ __forceinline__ void nt_stage_x_commit(uint16_t* __restrict__ lds16, const i32x4 (&v)[kNtXPer],
                                                  const NtParams& p, int k0, int span, int tid) {
    const int cpr = span / 8;
#pragma unroll
    for (int c = 0; c < kNtXPer; ++c) {
        const int i = tid + c * kThreads;
        if (i < cpr * MT) {
            const int m = i / cpr, q = i - m * cpr;
            const int kb = k0 + 8 * q;
            i32x4 w = v[c];
            if (kb + 8 > p.K) {                          // the chunk holding K: zero what lies past it
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t u = uint32_t(w[e]);
                    w[e] = int(((kb + 2 * e < p.K) ? (u & 0xFFFFu) : 0u) | ((kb + 2 * e + 1 < p.K) ? (u & 0xFFFF0000u) : 0u));
                }
            }
            if constexpr (MT == 1) {
                *reinterpret_cast<i32x4*>(lds16 + 8 * q) = w;
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    lds16[(8 * q + e) * MT + m] = static_cast<uint16_t>(uint32_t(w[e >> 1]) >> (16 * (e & 1)));
            }
        }
    }
}

// One wave's walk over its rows: G groups of R rows; step s is chunk j of every row of group g
// (s = g * J + j), so x's chunk is read from LDS once for R rows.  D steps are in flight
// (R * D loads per lane), and the step counter runs on across groups, so the loads of the
// next group's first chunks issue while the current group finishes.
template <int DT, int MT, int R, int D>
__global__ __launch_bounds__(kThreads) void gemv_nt_kernel(const NtParams p) {
    extern __shared__ float lds[];
    __shared__ int s_last;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bid = blockIdx.x;
    const int sl = bid % p.ks;
    const int rb = (bid / p.ks) % p.row_blocks;
    const int mb = bid / (p.ks * p.row_blocks);
    const int k0 = sl * p.slice_k;
    const int klen = min(p.slice_k, p.K - k0);
    const int J = (klen + kNtChunk - 1) / kNtChunk;     // wave-loads per row of the slice
    const int m0 = mb * MT;
    const int RW = 4 * p.r;                             // rows per workgroup
    const int G = p.r / R;                              // row groups per wave

    // ---- x[m0 : m0+MT, k0 : k0 + J*512] as 16-bit values in LDS, layout [k][m], zero past M and K
    uint16_t* lds16 = reinterpret_cast<uint16_t*>(lds);
    i32x4 xv[kNtXPer];
    nt_stage_x_issue<MT>(xv, p, m0, k0, J * kNtChunk, tid);

    const __amdgpu_buffer_rsrc_t wr = make_rsrc(p.wt, p.w_extent);
    const int row0 = rb * RW + wave * p.r;
    const int S = G * J;                                // steps of this wave
    // position of the next step to load (group lg, chunk lj, step ls), advanced without division
    int lg = 0, lj = 0, ls = 0;
    auto load_step = [&](i32x4 (&b)[R]) {
        const int k = k0 + lj * kNtChunk + 8 * lane;
#pragma unroll
        for (int i = 0; i < R; ++i) {
            const int n = row0 + lg * R + i;
            const uint32_t off = (ls < S && n < p.N && k < p.K) ? uint32_t(n) * p.row_bytes + uint32_t(k) * 2u : kOutOfRange;
            b[i] = __builtin_amdgcn_raw_buffer_load_b128(wr, off, 0, kLoadNT);
        }
        ++ls;
        if (++lj == J) {
            lj = 0;
            ++lg;
        }
    };
    i32x4 buf[D][R];
#pragma unroll
    for (int d = 0; d < D; ++d) load_step(buf[d]);
    nt_stage_x_commit<MT>(lds16, xv, p, k0, J * kNtChunk, tid);
    __syncthreads();

    const int64_t pbase = ((int64_t(mb) * p.row_blocks + rb) * p.ks + sl) * (int64_t(MT) * RW);
    const bool ragged_k = (p.K & 7) != 0;
    float acc[R][MT];
#pragma unroll
    for (int i = 0; i < R; ++i)
#pragma unroll
        for (int m = 0; m < MT; ++m) acc[i][m] = 0.f;
    int cg = 0, cj = 0;   // group and chunk of the step being consumed
    for (int s0 = 0; s0 < S; s0 += D) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
            if (s0 + d < S) {
                const int kb = cj * kNtChunk + 8 * lane;          // the lane's k within the slice
                float xr[8][MT];
                {
                    const i32x4* xs = reinterpret_cast<const i32x4*>(lds16 + kb * MT);
#pragma unroll
                    for (int c = 0; c < MT; ++c) {               // 8 * MT values: MT 16-byte reads
                        const i32x4 xc = xs[c];
#pragma unroll
                        for (int h = 0; h < 8; ++h) {
                            const int idx = 8 * c + h, e = idx / MT, m = idx - e * MT;
                            xr[e][m] = widen1<DT>(static_cast<uint16_t>(uint32_t(xc[h >> 1]) >> (16 * (h & 1))));
                        }
                    }
                }
                const bool mask = ragged_k && k0 + kb + 8 > p.K;   // padding past K must not reach the sums
#pragma unroll
                for (int i = 0; i < R; ++i) {
                    i32x4 v = buf[d][i];
                    if (mask) {
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const uint32_t w = uint32_t(v[q]);
                            const uint32_t lo = (k0 + kb + 2 * q < p.K) ? (w & 0xFFFFu) : 0u;
                            const uint32_t hi = (k0 + kb + 2 * q + 1 < p.K) ? (w & 0xFFFF0000u) : 0u;
                            v[q] = int(lo | hi);
                        }
                    }
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const uint32_t w = uint32_t(v[q]);
                        float lo, hi;
                        if constexpr (DT == NMM_BF16) {
                            lo = __uint_as_float(w << 16);
                            hi = __uint_as_float(w & 0xFFFF0000u);
                        } else {
                            const f16x2 h = __builtin_bit_cast(f16x2, w);
                            lo = static_cast<float>(h[0]);
                            hi = static_cast<float>(h[1]);
                        }
#pragma unroll
                        for (int m = 0; m < MT; ++m) {
                            acc[i][m] = __builtin_fmaf(lo, xr[2 * q][m], acc[i][m]);
                            acc[i][m] = __builtin_fmaf(hi, xr[2 * q + 1][m], acc[i][m]);
                        }
                    }
                }
                if (cj == J - 1) {                                // the group's rows are complete
#pragma unroll
                    for (int i = 0; i < R; ++i) {
                        const int n = row0 + cg * R + i;
#pragma unroll
                        for (int m = 0; m < MT; ++m) {
                            float v2 = acc[i][m];
                            v2 = add_ror<1>(v2);
                            v2 = add_ror<2>(v2);
                            v2 = add_ror<4>(v2);
                            v2 = add_ror<8>(v2);
                            v2 = add_xor16(v2);
                            v2 = add_xor32(v2);
                            acc[i][m] = 0.f;
                            if (lane == 0) {
                                if (p.ks == 1) {
                                    if (n < p.N && m0 + m < p.M) p.y[int64_t(m0 + m) * p.ldy + n] = v2;
                                } else {
                                    __hip_atomic_store(p.part + pbase + m * RW + wave * p.r + cg * R + i, v2,
                                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                                }
                            }
                        }
                    }
                    cj = 0;
                    ++cg;
                } else {
                    ++cj;
                }
            }
            load_step(buf[d]);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    if (p.ks == 1) return;
    // ---- split K: the row block's ticket; the last slice to arrive sums the slices in order
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) {
        s_last = arrive(p.tickets + int64_t(mb) * p.row_blocks + rb, unsigned(p.ks));
    }
    __syncthreads();
    if (!s_last) return;
    const int64_t gbase = (int64_t(mb) * p.row_blocks + rb) * p.ks * (int64_t(MT) * RW);
    for (int o = tid; o < MT * RW; o += kThreads) {
        const int m = o / RW, rr = o - m * RW;
        float sum = 0.f;
        for (int q = 0; q < p.ks; ++q)
            sum += __hip_atomic_load(p.part + gbase + int64_t(q) * (MT * RW) + o, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT);
        const int n = rb * RW + rr;
        if (n < p.N && m0 + m < p.M) p.y[int64_t(m0 + m) * p.ldy + n] = sum;
    }
}

// ---------------------------------------------------------------------------------------------
// MatMul 2 and the vector work behind it (Section IV-A, eq. 1-3): y = [c^KV | k^R] = h . W, then
// the cache entry [RMSNorm(c^KV) | RoPE(k^R, t)] in bf16.  The GEMV runs as above, except that
// y is stored device-coherently; every workgroup that writes the final outputs of a panel
// covering [c_off, c_off + kv + rope) counts the panel in on one counter, and the one that
// counts in last builds the entry from y.  No workgroup waits for another, so the launch cannot
// deadlock whatever else is resident.
// ---------------------------------------------------------------------------------------------
struct KvParams {
    const uint16_t* gamma;   // [kv] bf16 RMSNorm weight
    uint16_t* row;           // the cache row (bf16, kv + rope values)
    unsigned* done;          // the panel counter (zero before and after the launch)
    float eps;
    double freq_step;        // theta^(-2/rope): pair j turns freq_step^j radians per position
    int64_t position;
    int c_off, kv, rope, away;
    int first_panel, n_panels;   // the panels covering the entry's columns
};

constexpr double kTwoPiHi = 6.283185307179586;          // 2*pi rounded to double
constexpr double kTwoPiLo = 2.4492935982947064e-16;     // 2*pi - kTwoPiHi
constexpr double kInvTwoPi = 0.15915494309189535;

// Sine and cosine of RoPE pair j's angle a = t * theta^(-2j/rope) = t * freq_step^j.  The power
// is taken by binary powering and a formed in fp64 (relative error a few units of 2^-53), then a
// is reduced to [-pi, pi] by a two-term Cody-Waite step with fused multiply-adds (k * kTwoPiHi
// is exact for |k| < 2^30, i.e. positions below 2^31); the sine and cosine of the reduced angle
// are taken in fp32.
__device__ __forceinline__ void rope_angle(const KvParams& e, int j, float* sn, float* cs) {
    double f = 1.0, b = e.freq_step;
    for (int n = j; n; n >>= 1) {
        if (n & 1) f *= b;
        b *= b;
    }
    const double a = double(e.position) * f;
    const double k = rint(a * kInvTwoPi);
    const double r = fma(-k, kTwoPiLo, fma(-k, kTwoPiHi, a));
    sincosf(float(r), sn, cs);
}

// The entry from the product src[0 .. kv + rope) (written by this launch or an earlier one; the
// loads are device-coherent either way): src and gamma are staged in LDS in one pass (one round
// trip), then RMSNorm and RoPE (sn, cs: this thread's pair, taken earlier).
__device__ __forceinline__ void kv_entry(const float* src, const KvParams& e, float* lds, float sn, float cs) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n_all = e.kv + e.rope;
    float* vals = lds;                  // [n_all]
    float* gam = lds + n_all;           // [kv]
    float* red = gam + e.kv;            // [kWaves]
    float ss = 0.f;
    for (int i = tid; i < n_all; i += kThreads) {
        const float v = __hip_atomic_load(src + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        vals[i] = v;
        if (i < e.kv) {
            gam[i] = __uint_as_float(uint32_t(e.gamma[i]) << 16);
            ss += v * v;
        }
    }
    // mean of squares: a fixed butterfly inside each wave, then the waves in order
    ss = add_ror<1>(ss);
    ss = add_ror<2>(ss);
    ss = add_ror<4>(ss);
    ss = add_ror<8>(ss);
    ss = add_xor16(ss);
    ss = add_xor32(ss);
    if (lane == 0) red[wave] = ss;
    __syncthreads();
    float tot = red[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) tot += red[w];
    const float inv = 1.0f / __builtin_sqrtf(tot / float(e.kv) + e.eps);
    for (int i = tid; i < e.kv; i += kThreads) e.row[i] = to_bf16_mode(vals[i] * inv * gam[i], e.away);
    if (tid < e.rope / 2) {
        const float k0 = vals[e.kv + 2 * tid], k1 = vals[e.kv + 2 * tid + 1];
        e.row[e.kv + 2 * tid] = to_bf16_mode(k0 * cs - k1 * sn, e.away);
        e.row[e.kv + 2 * tid + 1] = to_bf16_mode(k0 * sn + k1 * cs, e.away);
    }
}

template <int U>
__global__ __launch_bounds__(kThreads) void gemv_kv_kernel(const KParams p, const KvParams e) {
    extern __shared__ float lds[];
    __shared__ int s_last;
    const int tid = threadIdx.x;
    const Item it = item_of<1>(p, blockIdx.x, tid);
    const bool counted = it.panel >= e.first_panel && it.panel < e.first_panel + e.n_panels;
    float acc[1][8];
    stream_item<NMM_BF16, 1, U>(p, it, lds, acc, tid);
    if (!counted) {
        reduce_item<1, kStorePlain>(p, it, acc, lds, tid);
        (void)finish_panel<1, kStorePlain>(p, it, &s_last, tid);
        return;
    }
    reduce_item<1, kStoreEpi>(p, it, acc, lds, tid);
    if (!finish_panel<1, kStoreEpi>(p, it, &s_last, tid)) return;
    // each workgroup that completes a panel takes the RoPE sines and cosines while its last
    // stores complete (the empty asm keeps the computation here); the last to count in uses them
    float sn = 0.f, cs = 1.f;
    if (tid < e.rope / 2) rope_angle(e, tid, &sn, &cs);
    asm volatile("" : "+v"(sn), "+v"(cs));
    // the panel's outputs are final: let their stores complete, then count the panel in
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) {
        s_last = arrive(e.done, unsigned(e.n_panels));
    }
    __syncthreads();
    if (s_last) kv_entry(p.y + e.c_off, e, lds, sn, cs);
}

// A batched GEMV launch (the per-head q_nope . W_UK of the absorbed query) with one extra
// workgroup, the last, that rotates each head's rope part of the query, q[h, nope : nope+rope]
// (fp32, from an earlier launch), and writes it as bf16 at q_out[h, kv : kv + rope].
struct QropeParams {
    const float* q;          // [heads, nope + rope] fp32
    uint16_t* q_out;         // [heads, ldq] bf16
    int64_t ldq;
    int heads, nope, kv;
};

template <int U>
__global__ __launch_bounds__(kThreads) void gemv_qrope_kernel(const KParams p, const KvParams e, const QropeParams r) {
    extern __shared__ float lds[];
    __shared__ int s_last;
    if (blockIdx.x == gridDim.x - 1) {
        const int pairs = e.rope / 2;
        if (pairs == 0) return;
        const int j = threadIdx.x % pairs, h0 = threadIdx.x / pairs, hstep = kThreads / pairs;
        if (h0 >= hstep) return;                     // threads past the last whole group of pairs
        float sn, cs;
        rope_angle(e, j, &sn, &cs);
        const int qk = r.nope + e.rope;
        for (int h = h0; h < r.heads; h += hstep) {
            const float k0 = r.q[int64_t(h) * qk + r.nope + 2 * j], k1 = r.q[int64_t(h) * qk + r.nope + 2 * j + 1];
            uint16_t* dst = r.q_out + int64_t(h) * r.ldq + r.kv + 2 * j;
            dst[0] = to_bf16_bits(k0 * cs - k1 * sn);
            dst[1] = to_bf16_bits(k0 * sn + k1 * cs);
        }
        return;
    }
    gemv_item<NMM_BF16, 1, U, kStorePlain>(p, blockIdx.x, lds, &s_last);
}

// A GEMV launch with one extra workgroup, the last, that builds the cache entry of a product an
// earlier launch on the stream completed (src).  The decode chain runs the entry of its
// down-projection this way beside W_UQ, so nothing on the chain waits for it.
template <int U>
__global__ __launch_bounds__(kThreads) void gemv_entry_kernel(const KParams p, const KvParams e, const float* src) {
    extern __shared__ float lds[];
    __shared__ int s_last;
    if (blockIdx.x == gridDim.x - 1) {
        float sn = 0.f, cs = 1.f;
        if (threadIdx.x < e.rope / 2) rope_angle(e, threadIdx.x, &sn, &cs);
        kv_entry(src, e, lds, sn, cs);
        return;
    }
    gemv_item<NMM_BF16, 1, U, kStorePlain>(p, blockIdx.x, lds, &s_last);
}

// y = 0 (and its bf16 copy) for K == 0: the empty sum.
__global__ void zero_output_kernel(float* y, int64_t ldy, int64_t sy, uint16_t* ybf, int64_t group,
                                   int64_t keep, int64_t ldm, int64_t sb, int64_t M, int64_t N,
                                   int64_t batch) {
    const int64_t total = batch * M * N;
    for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < total;
         i += int64_t(gridDim.x) * blockDim.x) {
        const int64_t n = i % N, m = (i / N) % M, b = i / (N * M);
        if (y) y[b * sy + m * ldy + n] = 0.f;
        if (ybf) {
            const int64_t g = n / group, r = n - g * group;
            if (r < keep) ybf[b * sb + m * ldm + g * keep + r] = 0;
        }
    }
}

__global__ void zero_bytes_kernel(uint8_t* p, size_t bytes) {
    const size_t n16 = bytes / 16;
    const size_t stride = size_t(gridDim.x) * blockDim.x;
    for (size_t i = blockIdx.x * size_t(blockDim.x) + threadIdx.x; i < n16; i += stride)
        reinterpret_cast<i32x4*>(p)[i] = i32x4{0, 0, 0, 0};
    for (size_t i = n16 * 16 + blockIdx.x * size_t(blockDim.x) + threadIdx.x; i < bytes; i += stride)
        p[i] = 0;
}

template <int DT, int MT, int U>
void launch_t(const KParams& kp, int64_t grid, size_t lds, hipStream_t s) {
    if (kp.y)
        hipLaunchKernelGGL((gemv_kernel<DT, MT, U, kStorePlain>), dim3(static_cast<uint32_t>(grid)), dim3(kThreads), lds, s, kp);
    else
        hipLaunchKernelGGL((gemv_kernel<DT, MT, U, kStoreNoY>), dim3(static_cast<uint32_t>(grid)), dim3(kThreads), lds, s, kp);
}

template <int DT, int MT>
void launch_u(const KParams& kp, int64_t grid, size_t lds, int unroll, hipStream_t s) {
    if constexpr (MT <= 2) {
        if (unroll == 16) {
            launch_t<DT, MT, 16>(kp, grid, lds, s);
            return;
        }
    }
    if (unroll == 8) launch_t<DT, MT, 8>(kp, grid, lds, s);
    else if (unroll == 4) launch_t<DT, MT, 4>(kp, grid, lds, s);
    else launch_t<DT, MT, 2>(kp, grid, lds, s);
}

template <int DT>
void launch_m(const KParams& kp, int64_t grid, size_t lds, int mt, int unroll, hipStream_t s) {
    switch (mt) {
        case 1: launch_u<DT, 1>(kp, grid, lds, unroll, s); break;
        case 2: launch_u<DT, 2>(kp, grid, lds, unroll, s); break;
        case 4: launch_u<DT, 4>(kp, grid, lds, unroll, s); break;
        case 8: launch_u<DT, 8>(kp, grid, lds, unroll, s); break;
        default: launch_u<DT, 16>(kp, grid, lds, unroll, s); break;
    }
}

nmm_status last_launch_status() {
    return hipGetLastError() == hipSuccess ? NMM_OK : NMM_ERR_HIP;
}

}  // namespace

nmm_status launch_zero_fill(void* ptr, size_t bytes, void* stream) {
    if (bytes == 0) return NMM_OK;
    const size_t blocks = std::min<size_t>(1024, (bytes / 16 + 255) / 256 + 1);
    hipLaunchKernelGGL(zero_bytes_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(256), 0,
                       static_cast<hipStream_t>(stream), static_cast<uint8_t*>(ptr), bytes);
    return last_launch_status();
}

namespace {

KParams make_params(const GemvArgs& a, const GemvPlan& p, unsigned* tickets, float* part) {
    KParams kp{};
    kp.x = static_cast<const uint16_t*>(a.x);
    kp.ldx = a.ldx;
    kp.sx = a.sx;
    kp.w = static_cast<const uint16_t*>(a.w);
    kp.sw = a.sw;
    kp.y = a.y;
    kp.ldy = a.ldy;
    kp.sy = a.sy;
    kp.ybf = static_cast<uint16_t*>(a.ybf);
    kp.ybf_group = a.ybf_group;
    kp.ybf_keep = a.ybf_keep;
    kp.ybf_ldm = a.ybf_ldm;
    kp.ybf_sb = a.ybf_sb;
    kp.ybf_away = a.ybf_away;
    kp.M = static_cast<int>(a.M);
    kp.K = static_cast<int>(a.K);
    kp.N = static_cast<int>(a.N);
    kp.row_bytes = static_cast<uint32_t>(a.ldw * 2);
    kp.w_extent = static_cast<uint32_t>(((a.K - 1) * a.ldw + (a.N + 7) / 8 * 8) * 2);
    kp.n_full = p.n_full;
    kp.tail_chunks = p.tail_chunks;
    auto log2i = [](int v) { int l = 0; while ((1 << l) < v) ++l; return l; };
    kp.full_lg = log2i(p.cw_full);
    kp.tail_lg = log2i(std::max(p.tail_cw, 1));
    kp.ks_full = p.ks_full;
    kp.rows_full = p.rows_full;
    kp.ks_tail = p.ks_tail;
    kp.rows_tail = p.rows_tail;
    kp.ks_max = p.ks_max;
    kp.items = p.items;
    kp.mblocks = p.mblocks;
    kp.n_panels = p.n_full + (p.tail_chunks ? 1 : 0);
    if (p.split()) {
        kp.tickets = tickets;
        kp.part = part;
    }
    return kp;
}

size_t gemv_lds_bytes(const GemvPlan& p) {
    const int rows_max = std::max(p.rows_full, p.rows_tail);
    const int mg = p.mt < 4 ? p.mt : 4;
    return std::max<size_t>(size_t(rows_max) * p.mt * 4, size_t(mg) * kThreads * 8 * 4);
}

}  // namespace

nmm_status launch_gemv(const GemvArgs& a, const GemvPlan& p, unsigned* tickets, float* part, void* stream) {
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (a.batch == 0 || a.M == 0 || a.N == 0) return NMM_OK;
    if (a.K == 0) {
        const int64_t total = a.batch * a.M * a.N;
        const int64_t blocks = std::min<int64_t>(4096, (total + 255) / 256);
        hipLaunchKernelGGL(zero_output_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(256), 0, s, a.y,
                           a.ldy, a.sy, static_cast<uint16_t*>(a.ybf), a.ybf_group, a.ybf_keep,
                           a.ybf_ldm, a.ybf_sb, a.M, a.N, a.batch);
        return last_launch_status();
    }
    const KParams kp = make_params(a, p, tickets, part);
    const size_t lds = gemv_lds_bytes(p);
    if (a.dt == NMM_BF16) launch_m<NMM_BF16>(kp, p.grid, lds, p.mt, p.unroll, s);
    else launch_m<NMM_F16>(kp, p.grid, lds, p.mt, p.unroll, s);
    return last_launch_status();
}

namespace {

// Whether the GEMV can share a launch with attention's or the merge's workgroups: bf16, one row,
// one batch entry, 8 or 16 row-steps in flight.
bool shareable(const GemvArgs& g, const GemvPlan& gp) {
    return g.dt == NMM_BF16 && g.batch == 1 && g.M == 1 && g.K > 0 && g.N > 0 && g.y && gp.mt == 1 &&
           (gp.unroll == 8 || gp.unroll == 16);
}

// The GEMV and attention's workgroups in one launch where both fit it (the 576 / 512 attention,
// the GEMV's LDS within one attention chunk buffer), else the two launches in order; no merge.
nmm_status gemv_beside_attention(const GemvArgs& g, const GemvPlan& gp, unsigned* tickets, float* part,
                                 const attn::AttnLaunch& al, hipStream_t s) {
    const bool fuse = al.grid > 0 && al.variant == attn::kAttnExact && al.p.pitch <= attn::kPitchMax &&
                      shareable(g, gp) && gemv_lds_bytes(gp) <= size_t(attn::kCh) * attn::kPitchMax * 2 &&
                      gp.grid + al.grid < (int64_t(1) << 31);
    if (!fuse) {
        nmm_status st = launch_gemv(g, gp, tickets, part, s);
        if (st != NMM_OK) return st;
        return launch_attention_kernel(al, s);
    }
    const KParams kp = make_params(g, gp, tickets, part);
    const dim3 grid(static_cast<uint32_t>(gp.grid + al.grid));
    if (gp.unroll == 16)
        hipLaunchKernelGGL(gemv_attention_kernel<16>, grid, dim3(kThreads), 0, s, kp, al.p, static_cast<uint32_t>(al.grid));
    else
        hipLaunchKernelGGL(gemv_attention_kernel<8>, grid, dim3(kThreads), 0, s, kp, al.p, static_cast<uint32_t>(al.grid));
    return last_launch_status();
}

}  // namespace

nmm_status launch_gemv_attention(const GemvArgs& g, const GemvPlan& gp, unsigned* tickets, float* part,
                                 const AttnArgs& a, void* attn_ws, size_t attn_ws_bytes, void* stream) {
    attn::AttnLaunch al;
    nmm_status st = prepare_attention(a, attn_ws, attn_ws_bytes, &al);
    if (st != NMM_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = gemv_beside_attention(g, gp, tickets, part, al, s);
    if (st != NMM_OK) return st;
    return launch_attention_merge(al, s);
}

nmm_status launch_gemv_beside_attention(const GemvArgs& g, const GemvPlan& gp, unsigned* tickets, float* part,
                                        const AttnArgs& a, void* attn_ws, size_t attn_ws_bytes, void* stream) {
    attn::AttnLaunch al;
    nmm_status st = prepare_attention(a, attn_ws, attn_ws_bytes, &al);
    if (st != NMM_OK) return st;
    return gemv_beside_attention(g, gp, tickets, part, al, static_cast<hipStream_t>(stream));
}

nmm_status launch_gemv_merge(const GemvArgs& g, const GemvPlan& gp, unsigned* tickets, float* part,
                             const AttnArgs& a, void* attn_ws, size_t attn_ws_bytes, void* stream) {
    attn::AttnLaunch al;
    nmm_status st = prepare_attention(a, attn_ws, attn_ws_bytes, &al);
    if (st != NMM_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (al.merge_grid == 0 || !shareable(g, gp)) {
        st = launch_gemv(g, gp, tickets, part, stream);
        if (st != NMM_OK) return st;
        return launch_attention_merge(al, s);
    }
    // one workgroup per merge block: they take the compute units the GEMV leaves free and share
    // the others with its workgroups (no LDS of their own), so each waits only for its own loads
    // -- under the GEMV's weight stream a memory round trip takes microseconds
    const int64_t extra = al.merge_grid;
    const KParams kp = make_params(g, gp, tickets, part);
    const dim3 grid(static_cast<uint32_t>(gp.grid + extra));
    const size_t lds = gemv_lds_bytes(gp);
    const uint32_t gg = static_cast<uint32_t>(gp.grid), mb = static_cast<uint32_t>(al.merge_grid);
    if (gp.unroll == 16) hipLaunchKernelGGL(gemv_merge_kernel<16>, grid, dim3(kThreads), lds, s, kp, al.p, gg, mb);
    else hipLaunchKernelGGL(gemv_merge_kernel<8>, grid, dim3(kThreads), lds, s, kp, al.p, gg, mb);
    return last_launch_status();
}

namespace {

KvParams make_kv_params(const GemvPlan& p, const KvEpilogue& e) {
    KvParams kv{};
    kv.gamma = static_cast<const uint16_t*>(e.gamma);
    kv.row = static_cast<uint16_t*>(e.row);
    kv.done = e.done;
    kv.eps = e.eps;
    kv.freq_step = e.rope > 0 ? std::pow(double(e.theta), -2.0 / double(e.rope)) : 1.0;
    kv.position = e.position;
    kv.c_off = static_cast<int>(e.c_off);
    kv.kv = e.kv;
    kv.rope = e.rope;
    kv.away = e.away;
    const int64_t pcols = int64_t(p.cw_full) * 8;
    kv.first_panel = static_cast<int>(e.c_off / pcols);
    kv.n_panels = static_cast<int>((e.c_off + e.kv + e.rope - 1) / pcols) - kv.first_panel + 1;
    return kv;
}

}  // namespace

nmm_status launch_gemv_nt(const GemvArgs& a, const NtPlan& p, unsigned* tickets, float* part, void* stream) {
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (a.M == 0 || a.N == 0) return NMM_OK;
    if (a.K == 0) {
        const int64_t total = a.M * a.N;
        const int64_t blocks = std::min<int64_t>(4096, (total + 255) / 256);
        hipLaunchKernelGGL(zero_output_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(256), 0, s, a.y, a.ldy,
                           int64_t(0), static_cast<uint16_t*>(nullptr), int64_t(1), int64_t(1), int64_t(0), int64_t(0),
                           a.M, a.N, int64_t(1));
        return last_launch_status();
    }
    NtParams np{};
    np.x = static_cast<const uint16_t*>(a.x);
    np.ldx = a.ldx;
    np.wt = static_cast<const uint16_t*>(a.w);
    np.row_bytes = static_cast<uint32_t>(a.ldw * 2);
    np.w_extent = static_cast<uint32_t>(((a.N - 1) * a.ldw + (a.K + 7) / 8 * 8) * 2);
    np.y = a.y;
    np.ldy = a.ldy;
    np.part = part;
    np.tickets = tickets;
    np.M = static_cast<int>(a.M);
    np.K = static_cast<int>(a.K);
    np.N = static_cast<int>(a.N);
    np.r = p.r;
    np.slice_k = p.slice_k;
    np.ks = p.ks;
    np.row_blocks = p.row_blocks;
    np.mblocks = p.mblocks;
    const size_t lds = size_t(p.slice_k) * p.mt * 2;
    const dim3 grid(static_cast<uint32_t>(p.grid)), block(kThreads);
#define NMM_NT_LAUNCH(DTV, MTV)                                                                                  \
    do {                                                                                                         \
        switch (p.rgroup) {                                                                                      \
            case 8: hipLaunchKernelGGL((gemv_nt_kernel<DTV, MTV, 8, 1>), grid, block, lds, s, np); break;        \
            case 4: hipLaunchKernelGGL((gemv_nt_kernel<DTV, MTV, 4, 2>), grid, block, lds, s, np); break;        \
            case 2: hipLaunchKernelGGL((gemv_nt_kernel<DTV, MTV, 2, 4>), grid, block, lds, s, np); break;        \
            default: hipLaunchKernelGGL((gemv_nt_kernel<DTV, MTV, 1, 8>), grid, block, lds, s, np); break;       \
        }                                                                                                        \
    } while (0)
#define NMM_NT_LAUNCH16(DTV)                                                                                     \
    do {                                                                                                         \
        switch (p.rgroup) {                                                                                      \
            case 8: hipLaunchKernelGGL((gemv_nt_kernel<DTV, 1, 8, 2>), grid, block, lds, s, np); break;          \
            case 4: hipLaunchKernelGGL((gemv_nt_kernel<DTV, 1, 4, 4>), grid, block, lds, s, np); break;          \
            case 2: hipLaunchKernelGGL((gemv_nt_kernel<DTV, 1, 2, 8>), grid, block, lds, s, np); break;          \
            default: hipLaunchKernelGGL((gemv_nt_kernel<DTV, 1, 1, 16>), grid, block, lds, s, np); break;        \
        }                                                                                                        \
    } while (0)
    if (p.depth == 16) {
        if (a.dt == NMM_BF16) NMM_NT_LAUNCH16(NMM_BF16);
        else NMM_NT_LAUNCH16(NMM_F16);
    } else if (a.dt == NMM_BF16) {
        if (p.mt == 1) NMM_NT_LAUNCH(NMM_BF16, 1);
        else if (p.mt == 2) NMM_NT_LAUNCH(NMM_BF16, 2);
        else NMM_NT_LAUNCH(NMM_BF16, 4);
    } else {
        if (p.mt == 1) NMM_NT_LAUNCH(NMM_F16, 1);
        else if (p.mt == 2) NMM_NT_LAUNCH(NMM_F16, 2);
        else NMM_NT_LAUNCH(NMM_F16, 4);
    }
#undef NMM_NT_LAUNCH
#undef NMM_NT_LAUNCH16
    return last_launch_status();
}

nmm_status launch_gemv_kv(const GemvArgs& a, const GemvPlan& p, unsigned* tickets, float* part,
                          const KvEpilogue& e, void* stream) {
    hipStream_t s = static_cast<hipStream_t>(stream);
    const KParams kp = make_params(a, p, tickets, part);
    const KvParams kv = make_kv_params(p, e);
    const size_t lds = gemv_kv_lds_bytes(p, e.kv, e.rope);
    const dim3 grid(static_cast<uint32_t>(p.grid)), block(kThreads);
    switch (p.unroll) {
        case 16: hipLaunchKernelGGL(gemv_kv_kernel<16>, grid, block, lds, s, kp, kv); break;
        case 8: hipLaunchKernelGGL(gemv_kv_kernel<8>, grid, block, lds, s, kp, kv); break;
        case 4: hipLaunchKernelGGL(gemv_kv_kernel<4>, grid, block, lds, s, kp, kv); break;
        default: hipLaunchKernelGGL(gemv_kv_kernel<2>, grid, block, lds, s, kp, kv); break;
    }
    return last_launch_status();
}

nmm_status launch_gemv_entry(const GemvArgs& a, const GemvPlan& p, unsigned* tickets, float* part,
                             const KvEpilogue& e, const float* src, void* stream) {
    hipStream_t s = static_cast<hipStream_t>(stream);
    const KParams kp = make_params(a, p, tickets, part);
    const KvParams kv = make_kv_params(p, e);
    const size_t lds = gemv_kv_lds_bytes(p, e.kv, e.rope);
    const dim3 grid(static_cast<uint32_t>(p.grid + 1)), block(kThreads);
    switch (p.unroll) {
        case 16: hipLaunchKernelGGL(gemv_entry_kernel<16>, grid, block, lds, s, kp, kv, src); break;
        case 8: hipLaunchKernelGGL(gemv_entry_kernel<8>, grid, block, lds, s, kp, kv, src); break;
        case 4: hipLaunchKernelGGL(gemv_entry_kernel<4>, grid, block, lds, s, kp, kv, src); break;
        default: hipLaunchKernelGGL(gemv_entry_kernel<2>, grid, block, lds, s, kp, kv, src); break;
    }
    return last_launch_status();
}

nmm_status launch_gemv_qrope(const GemvArgs& a, const GemvPlan& p, unsigned* tickets, float* part, const float* q,
                             void* q_out, int64_t ldq, int heads, int nope, int kv, int rope, int64_t position,
                             float theta, void* stream) {
    hipStream_t s = static_cast<hipStream_t>(stream);
    const KParams kp = make_params(a, p, tickets, part);
    KvEpilogue e;
    e.theta = theta;
    e.position = position;
    e.rope = rope;
    const KvParams kv_p = make_kv_params(p, e);
    QropeParams r{};
    r.q = q;
    r.q_out = static_cast<uint16_t*>(q_out);
    r.ldq = ldq;
    r.heads = heads;
    r.nope = nope;
    r.kv = kv;
    const size_t lds = gemv_lds_bytes(p);
    const dim3 grid(static_cast<uint32_t>(p.grid + 1)), block(kThreads);
    switch (p.unroll) {
        case 16: hipLaunchKernelGGL(gemv_qrope_kernel<16>, grid, block, lds, s, kp, kv_p, r); break;
        case 8: hipLaunchKernelGGL(gemv_qrope_kernel<8>, grid, block, lds, s, kp, kv_p, r); break;
        case 4: hipLaunchKernelGGL(gemv_qrope_kernel<4>, grid, block, lds, s, kp, kv_p, r); break;
        default: hipLaunchKernelGGL(gemv_qrope_kernel<2>, grid, block, lds, s, kp, kv_p, r); break;
    }
    return last_launch_status();
}

size_t gemv_kv_lds_bytes(const GemvPlan& p, int kv, int rope) {
    return std::max(gemv_lds_bytes(p), size_t(2 * kv + rope + kWaves) * 4);
}

namespace {

// ---------------------------------------------------------------------------------------------
// The decode chain's per-head pair W_UK -> W_UV in one launch (bf16, M = 1).  Head h's two
// products depend only on each other, so one workgroup runs both:
//   lat_h = q_nope_h . W_UK[h]  ([nope] x [nope, 512]),  lat'_h = bf16(lat_h)
//   o_h   = lat'_h . W_UV[h]    ([512] x [512, 128]),    o'_h   = bf16(o_h)
// It streams W_UK[h] and then W_UV[h] as one sequence of row-steps with U steps in flight, so
// W_UV's first loads are out while W_UK's sums are reduced; no second launch, no split-K.
// With NW waves (8 where nope allows it, else 4):
//  * W_UK step t: wave w reads row NW t + w (1 KB, 16 bytes per lane).
//  * W_UV step t: wave w reads rows 4 NW t + 4w .. + 3 (256 bytes each, 16 lanes per row).
// One workgroup per head covers half the device, so its bytes in flight decide the rate: 8 waves
// of 16 row-steps keep all of W_UK[h] (128 KB at nope 128) in flight at once.
// ---------------------------------------------------------------------------------------------
constexpr int kPairLat = 512;     // kv_lora
constexpr int kPairV = 128;       // v_head
constexpr int kPairMaxNope = 512;

struct PairParams {
    const uint16_t* q;    // q_nope bf16, head h at q + h * sq
    int64_t sq;
    const uint16_t* wuk;  // [heads][nope][512]
    const uint16_t* wuv;  // [heads][512][128]
    float* lat;           // [heads][512]
    uint16_t* latb;
    float* o;             // [heads][128]
    uint16_t* ob;
    int nope;
};

template <int U, int NW>
__device__ __forceinline__ void head_pair_block(const PairParams& p, int64_t h) {
    __shared__ __attribute__((aligned(16))) float xs[kPairMaxNope];   // q_nope of the head
    __shared__ __attribute__((aligned(16))) float red[NW * kPairLat];
    __shared__ float lat_s[kPairLat];                                 // lat'_h, widened
    constexpr int kT = 64 * NW;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int ta = p.nope / NW;                         // W_UK row-steps (a multiple of U)
    constexpr int kTb = kPairLat / (4 * NW);            // W_UV row-steps
    const __amdgpu_buffer_rsrc_t uk =
        make_rsrc(p.wuk + h * int64_t(p.nope) * kPairLat, uint32_t(p.nope) * kPairLat * 2);
    const __amdgpu_buffer_rsrc_t uv = make_rsrc(p.wuv + h * int64_t(kPairLat) * kPairV, kPairLat * kPairV * 2);
    auto off_a = [&](int t) { return uint32_t((NW * t + wave) * (kPairLat * 2) + lane * 16); };
    auto off_b = [&](int t) {
        return t < kTb ? uint32_t((4 * NW * t + 4 * wave + (lane >> 4)) * (kPairV * 2) + (lane & 15) * 16) : kOutOfRange;
    };

    // q_nope_h first (8 values per lane), then the first U row-steps, then q to LDS
    i32x4 qv = __builtin_amdgcn_raw_buffer_load_b128(make_rsrc(p.q + h * p.sq, uint32_t(p.nope) * 2),
                                                    tid * 8 < p.nope ? uint32_t(tid * 16) : kOutOfRange, 0, 0);
    i32x4 buf[U];
#pragma unroll
    for (int u = 0; u < U; ++u) buf[u] = __builtin_amdgcn_raw_buffer_load_b128(uk, off_a(u), 0, kLoadNT);
    if (tid * 8 < p.nope) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t w = static_cast<uint32_t>(qv[i]);
            xs[tid * 8 + 2 * i] = __uint_as_float(w << 16);
            xs[tid * 8 + 2 * i + 1] = __uint_as_float(w & 0xFFFF0000u);
        }
    }
    __syncthreads();

    // ---- lat_h: row 4t + wave, columns 8 lane .. + 7
    float acc[1][8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[0][e] = 0.f;
    int t0 = 0;
    for (; t0 + U < ta; t0 += U) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            fma_chunk<NMM_BF16, 1>(acc, buf[u], xs + NW * (t0 + u) + wave);
            buf[u] = __builtin_amdgcn_raw_buffer_load_b128(uk, off_a(t0 + u + U), 0, kLoadNT);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {   // the last U steps reload with W_UV's first U
        fma_chunk<NMM_BF16, 1>(acc, buf[u], xs + NW * (t0 + u) + wave);
        buf[u] = __builtin_amdgcn_raw_buffer_load_b128(uv, off_b(u), 0, kLoadNT);
        __builtin_amdgcn_sched_barrier(0);
    }
    // the waves' row sums, in wave order; lat and its bf16 rounding out, lat' to LDS
    *reinterpret_cast<f32x4*>(red + wave * kPairLat + 8 * lane) = f32x4{acc[0][0], acc[0][1], acc[0][2], acc[0][3]};
    *reinterpret_cast<f32x4*>(red + wave * kPairLat + 8 * lane + 4) = f32x4{acc[0][4], acc[0][5], acc[0][6], acc[0][7]};
    lds_barrier();
    for (int c = tid; c < kPairLat; c += kT) {
        float v = red[c];
#pragma unroll
        for (int w = 1; w < NW; ++w) v += red[w * kPairLat + c];
        const uint16_t b = to_bf16_bits(v);
        p.lat[h * kPairLat + c] = v;
        p.latb[h * kPairLat + c] = b;
        lat_s[c] = __uint_as_float(uint32_t(b) << 16);
    }
    lds_barrier();

    // ---- o_h: rows 4 NW t + 4 wave + lane / 16, columns 8 (lane % 16) .. + 7
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[0][e] = 0.f;
    const int rsub = 4 * wave + (lane >> 4);
    for (int t = 0; t < kTb; t += U) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            fma_chunk<NMM_BF16, 1>(acc, buf[u], lat_s + 4 * NW * (t + u) + rsub);
            buf[u] = __builtin_amdgcn_raw_buffer_load_b128(uv, off_b(t + u + U), 0, kLoadNT);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    // fold the wave's four row groups (lanes c, c + 16, c + 32, c + 48), then the waves in order
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[0][e] = add_xor32(add_xor16(acc[0][e]));
    if (lane < 16) {
        *reinterpret_cast<f32x4*>(red + wave * kPairV + 8 * lane) = f32x4{acc[0][0], acc[0][1], acc[0][2], acc[0][3]};
        *reinterpret_cast<f32x4*>(red + wave * kPairV + 8 * lane + 4) = f32x4{acc[0][4], acc[0][5], acc[0][6], acc[0][7]};
    }
    lds_barrier();
    if (tid < kPairV) {
        float v = red[tid];
#pragma unroll
        for (int w = 1; w < NW; ++w) v += red[w * kPairV + tid];
        p.o[h * kPairV + tid] = v;
        p.ob[h * kPairV + tid] = to_bf16_bits(v);
    }
}

template <int U, int NW>
__global__ __launch_bounds__(64 * NW) void head_pair_kernel(const PairParams p) {
    head_pair_block<U, NW>(p, blockIdx.x);
}

// The pair with the merge of an attention launched earlier: workgroups [0, heads) are the pair's,
// the rest run merge_block's 256-thread blocks (64 NW / 256 per workgroup) in turn.  The pair's
// one workgroup per head leaves compute units free, and the merge reads only the attention's span
// partials, so it runs beside the pair instead of under a later GEMV's weight stream.
template <int U, int NW>
__global__ __launch_bounds__(64 * NW) void head_pair_merge_kernel(const PairParams p, const attn::AttnParams a,
                                                                  uint32_t heads, uint32_t merge_blocks) {
    static_assert((64 * NW) % attn::kMergeThreads == 0, "whole merge blocks per workgroup");
    if (blockIdx.x < heads) {
        head_pair_block<U, NW>(p, blockIdx.x);
        return;
    }
    constexpr uint32_t kSub = 64 * NW / attn::kMergeThreads;
    const uint32_t sub = threadIdx.x / attn::kMergeThreads, t = threadIdx.x % attn::kMergeThreads;
    const uint32_t n = (gridDim.x - heads) * kSub;
    for (uint32_t b = (blockIdx.x - heads) * kSub + sub; b < merge_blocks; b += n)
        attn::merge_block(a, static_cast<int>(b), static_cast<int>(t));
}

PairParams pair_params(int64_t nope, const void* q_nope, const void* w_uk, const void* w_uv, float* lat,
                       void* lat_bf16, float* o, void* o_bf16) {
    PairParams pp{};
    pp.q = static_cast<const uint16_t*>(q_nope);
    pp.sq = nope;
    pp.wuk = static_cast<const uint16_t*>(w_uk);
    pp.wuv = static_cast<const uint16_t*>(w_uv);
    pp.lat = lat;
    pp.latb = static_cast<uint16_t*>(lat_bf16);
    pp.o = o;
    pp.ob = static_cast<uint16_t*>(o_bf16);
    pp.nope = static_cast<int>(nope);
    return pp;
}

}  // namespace

bool head_pair_ok(int64_t heads, int64_t nope, int64_t kv_lora, int64_t v_head) {
    return heads >= 1 && heads < (int64_t(1) << 31) && kv_lora == kPairLat && v_head == kPairV && nope >= 4 * kPairUnroll &&
           nope <= kPairMaxNope && nope % (4 * kPairUnroll) == 0;
}

nmm_status launch_head_pair(int64_t heads, int64_t nope, const void* q_nope, const void* w_uk, const void* w_uv,
                            float* lat, void* lat_bf16, float* o, void* o_bf16, void* stream) {
    const PairParams pp = pair_params(nope, q_nope, w_uk, w_uv, lat, lat_bf16, o, o_bf16);
    if (nope % (8 * kPairUnroll) == 0)
        hipLaunchKernelGGL((head_pair_kernel<kPairUnroll, 8>), dim3(static_cast<uint32_t>(heads)), dim3(8 * 64), 0,
                           static_cast<hipStream_t>(stream), pp);
    else
        hipLaunchKernelGGL((head_pair_kernel<kPairUnroll, 4>), dim3(static_cast<uint32_t>(heads)), dim3(4 * 64), 0,
                           static_cast<hipStream_t>(stream), pp);
    return last_launch_status();
}

nmm_status launch_head_pair_merge(int64_t heads, int64_t nope, const void* q_nope, const void* w_uk, const void* w_uv,
                                  float* lat, void* lat_bf16, float* o, void* o_bf16, const AttnArgs& a,
                                  void* attn_ws, size_t attn_ws_bytes, void* stream) {
    attn::AttnLaunch al;
    nmm_status st = prepare_attention(a, attn_ws, attn_ws_bytes, &al);
    if (st != NMM_OK) return st;
    if (al.merge_grid == 0) return launch_head_pair(heads, nope, q_nope, w_uk, w_uv, lat, lat_bf16, o, o_bf16, stream);
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (heads + al.merge_grid >= (int64_t(1) << 31)) {
        st = launch_head_pair(heads, nope, q_nope, w_uk, w_uv, lat, lat_bf16, o, o_bf16, stream);
        if (st != NMM_OK) return st;
        return launch_attention_merge(al, s);
    }
    const PairParams pp = pair_params(nope, q_nope, w_uk, w_uv, lat, lat_bf16, o, o_bf16);
    const uint32_t h = static_cast<uint32_t>(heads), mb = static_cast<uint32_t>(al.merge_grid);
    // one workgroup per merge block pair (or block, with 4 waves): they take the compute units the
    // pair leaves free
    if (nope % (8 * kPairUnroll) == 0) {
        const uint32_t extra = (mb + 1) / 2;
        hipLaunchKernelGGL((head_pair_merge_kernel<kPairUnroll, 8>), dim3(h + extra), dim3(8 * 64), 0, s, pp, al.p, h, mb);
    } else {
        hipLaunchKernelGGL((head_pair_merge_kernel<kPairUnroll, 4>), dim3(h + mb), dim3(4 * 64), 0, s, pp, al.p, h, mb);
    }
    return last_launch_status();
}

}  // namespace nmm
