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
#include <cstdint>
#include <cstdlib>

#include "nmm_internal.h"

namespace nmm {
namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
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
// flight: the load for step s+U is issued right after step s's data is taken.  The steady-state
// loop has no branches, so the compiler's wait counters track each load individually.
template <int DT, int MT, int U, bool GUARD>
__device__ __forceinline__ void stream_rows(float (&acc)[MT][8], i32x4 (&buf)[U], const Stream& st,
                                            int nsteps, const float* __restrict__ xs, int xs_step) {
    int s = 0;
    for (; s + U < nsteps; s += U) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const i32x4 cur = buf[u];
            const int sn = s + U + u;
            buf[u] = load_chunk<GUARD>(st.rsrc, st.off + sn * st.step_bytes, st.row + sn * st.rstep < st.K);
            fma_chunk<DT, MT>(acc, cur, xs + (s + u) * xs_step);
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) fma_chunk<DT, MT>(acc, buf[u], xs + (s + u) * xs_step);
}

__device__ __forceinline__ uint16_t to_bf16_bits(float v) {
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(v));
}

// Cache policy of x loads inside the fused chain: device-coherent (sc1), because x was written
// by other workgroups of the same launch and this XCD's L2 may hold older copies.
constexpr int kLoadCoherent = 16;

// y[m, n] (fp32) and its optional bf16 copy.  Inside the fused chain the bf16 copy is the next
// MatMul's operand, read by other workgroups during the same launch, so it is written with a
// device-scope atomic store (coherent at memory).
template <bool CHAIN>
__device__ __forceinline__ void store_out(const KParams& p, int64_t b, int m, int n, float v) {
    p.y[b * p.sy + int64_t(m) * p.ldy + n] = v;
    if (p.ybf) {
        const int64_t g = n / p.ybf_group, r = n - g * p.ybf_group;
        if (r < p.ybf_keep) {
            uint16_t* dst = p.ybf + b * p.ybf_sb + int64_t(m) * p.ybf_ldm + g * p.ybf_keep + r;
            if constexpr (CHAIN) __hip_atomic_store(dst, to_bf16_bits(v), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            else *dst = to_bf16_bits(v);
        }
    }
}

// Stage x[m0:m0+MT, k0:k0+rows] into LDS as fp32, layout [row][m], zero outside M x K.  Each
// thread fetches 16-byte chunks of x rows (8 consecutive k); every chunk load is issued before
// any is used, and chunks past x's extent read as zeros.
template <int DT, int MT, int AUX>
__device__ __forceinline__ void stage_x(float* __restrict__ lds, const KParams& p, int64_t b, int m0,
                                        int k0, int rows, int tid) {
    const int cpr = rows / 8;                       // chunks per x row of the slice
    const int total = cpr * MT;
    const int mrows = min(MT, p.M - m0);
    // x's extent reaches the 16-byte chunk holding each row's last element (ABI rule)
    const uint32_t x_extent = uint32_t(((int64_t(m0) + mrows - 1) * p.ldx + (p.K + 7) / 8 * 8) * 2);
    const __amdgpu_buffer_rsrc_t xr = make_rsrc(p.x + b * p.sx, x_extent);
    constexpr int kMaxPer = (kXStageBytes / 4 / 8 + kThreads - 1) / kThreads;   // chunks per thread
    i32x4 v[kMaxPer];
#pragma unroll
    for (int j = 0; j < kMaxPer; ++j) {
        const int i = tid + j * kThreads;
        const int m = i / cpr, q = i - m * cpr;
        const bool ok = i < total && m < mrows;
        const uint32_t off = ok ? uint32_t(((int64_t(m0) + m) * p.ldx + k0 + 8 * q) * 2) : kOutOfRange;
        v[j] = __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, AUX);
    }
#pragma unroll
    for (int j = 0; j < kMaxPer; ++j) {
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

// The fused chain's cross-workgroup dependency: the items of a MatMul may only read its x once
// the previous MatMul has finished all of its panels.
struct Dep {
    unsigned* wait_on = nullptr;   // completed-panel counter of the producing MatMul (or null)
    unsigned target = 0;           // its panel count
    unsigned* done = nullptr;      // this MatMul's completed-panel counter
    unsigned* error = nullptr;     // set when a wait gives up
    int spin_limit = 0;
    int sleep_reps = 1;            // s_sleep(2) repetitions between polls
};

// Wait until *d.wait_on reaches d.target.  Bounded: after spin_limit polls the wait gives up
// and raises the error flag, so a broken dependency can never hang the GPU.
__device__ __forceinline__ void wait_dependency(const Dep& d) {
    if (threadIdx.x == 0) {
        int spins = 0;
        while (__hip_atomic_load(d.wait_on, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < d.target) {
            if (++spins > d.spin_limit) {
                __hip_atomic_store(d.error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                break;
            }
            for (int r = 0; r < d.sleep_reps; ++r) __builtin_amdgcn_s_sleep(2);
        }
    }
    __syncthreads();
}

// Count one more completed panel, after every thread's output stores have completed.
__device__ __forceinline__ void signal_done(const Dep& d) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) __hip_atomic_fetch_add(d.done, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// One work item: one K-slice of one panel of one (batch entry, row block).  `bid` is the item's
// index within its MatMul.  CHAIN adds the fused chain's dependency wait and completion signal.
template <int DT, int MT, int U, bool CHAIN>
__device__ __forceinline__ void gemv_item(const KParams& p, uint32_t bid, float* lds, int* s_last, const Dep& dep) {
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;

    const int item = static_cast<int>(bid % uint32_t(p.items));
    const uint32_t bm = bid / uint32_t(p.items);
    const int mb = static_cast<int>(bm % uint32_t(p.mblocks));
    const int64_t b = bm / uint32_t(p.mblocks);

    // which panel and K-slice this workgroup owns
    int panel, slice, lg, ks, rows, valid;
    if (item < p.n_full * p.ks_full) {
        panel = item / p.ks_full;
        slice = item - panel * p.ks_full;
        lg = p.full_lg;
        ks = p.ks_full;
        rows = p.rows_full;
        valid = 1 << p.full_lg;
    } else {
        panel = p.n_full;
        slice = item - p.n_full * p.ks_full;
        lg = p.tail_lg;
        ks = p.ks_tail;
        rows = p.rows_tail;
        valid = p.tail_chunks;
    }
    const int cw = 1 << lg;                 // lanes across the panel's columns
    const int c = lane & (cw - 1);
    const int rstep = kWaves << (6 - lg);   // rows per workgroup step
    const int rin = wave * (64 >> lg) + (lane >> lg);
    const int k0 = slice * rows;
    const int m0 = mb * MT;
    const int chunk0 = panel << p.full_lg;  // first 8-column chunk of the panel
    const bool guard = k0 + rows > p.K;     // only the last K-slice reaches past K

    // ---- init: issue the first U loads of W (they do not depend on x), then stage x
    Stream st;
    {
        const int cc = c < valid ? c : valid - 1;   // lanes past a ragged edge re-read its last chunk
        st.rsrc = make_rsrc(p.w + b * p.sw, p.w_extent);
        st.off = uint32_t(k0 + rin) * p.row_bytes + uint32_t(chunk0 + cc) * 16u;
        st.step_bytes = uint32_t(rstep) * p.row_bytes;
        st.row = k0 + rin;
        st.rstep = rstep;
        st.K = p.K;
    }
    i32x4 buf[U];
    if (guard) prefetch<U, true>(buf, st);
    else prefetch<U, false>(buf, st);
    if constexpr (CHAIN) {
        if (dep.wait_on) {
            wait_dependency(dep);
            stage_x<DT, MT, kLoadCoherent>(lds, p, b, m0, k0, rows, tid);
        } else {
            stage_x<DT, MT, 0>(lds, p, b, m0, k0, rows, tid);
        }
    } else {
        stage_x<DT, MT, 0>(lds, p, b, m0, k0, rows, tid);
    }
    __syncthreads();

    // ---- compute: stream this workgroup's rows of the panel
    float acc[MT][8];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[m][j] = 0.f;
    {
        const int nsteps = rows / rstep;
        const float* xs = lds + rin * MT;
        if (guard) stream_rows<DT, MT, U, true>(acc, buf, st, nsteps, xs, rstep * MT);
        else stream_rows<DT, MT, U, false>(acc, buf, st, nsteps, xs, rstep * MT);
    }
    __syncthreads();   // x slice no longer needed: LDS becomes the reduction buffer

    // ---- gather, part 1: reduce the workgroup's row groups (fixed order) per m-group
    constexpr int MG = MT < 4 ? MT : 4;
    const int pcols = cw * 8;                                  // columns of this panel
    const int64_t pbase = (((b * p.mblocks + mb) * p.n_panels + panel) * int64_t(p.ks_max)) *
                          (int64_t(MT) * kPanelCols);
#pragma unroll
    for (int g = 0; g < MT; g += MG) {
#pragma unroll
        for (int mm = 0; mm < MG; ++mm) {
            float* dst = lds + ((mm * rstep + rin) * cw + c) * 8;
            *reinterpret_cast<f32x4*>(dst) = f32x4{acc[g + mm][0], acc[g + mm][1], acc[g + mm][2], acc[g + mm][3]};
            *reinterpret_cast<f32x4*>(dst + 4) = f32x4{acc[g + mm][4], acc[g + mm][5], acc[g + mm][6], acc[g + mm][7]};
        }
        __syncthreads();
        for (int o = tid; o < MG * pcols; o += kThreads) {
            const int mm = o / pcols, col = o - mm * pcols;
            float s = 0.f;
            for (int r = 0; r < rstep; ++r) s += lds[(mm * rstep + r) * pcols + col];
            const int m = g + mm;
            const int n = chunk0 * 8 + col;
            if (ks == 1) {
                if (m0 + m < p.M && n < p.N) store_out<CHAIN>(p, b, m0 + m, n, s);
            } else {
                __hip_atomic_store(p.part + pbase + int64_t(slice) * (MT * kPanelCols) + m * kPanelCols + col,
                                   s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        __syncthreads();
    }
    if (ks == 1) {
        if constexpr (CHAIN) signal_done(dep);
        return;
    }

    // ---- gather, part 2: the last workgroup of this panel sums the K-slices in order.
    // The partial sums above were written with device-scope atomic stores, which the GPU makes
    // coherent at memory (past the per-XCD L2 caches); the ticket is a device-scope atomic too,
    // and the last workgroup reads the partials with device-scope atomic loads.  Waiting for
    // every store to complete (s_waitcnt 0) before the ticket increment, and for the ticket's
    // value before the loads, orders the hand-off without writing back or invalidating the L2.
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) {
        unsigned* t = p.tickets + (b * p.mblocks + mb) * p.n_panels + panel;
        const unsigned prev = __hip_atomic_fetch_add(t, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const int last = prev == unsigned(ks - 1);
        if (last) __hip_atomic_store(t, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *s_last = last;
    }
    __syncthreads();
    if (!*s_last) return;
    // every output of the panel sums its slices in slice order; the loads of R outputs x QB
    // slices are all in flight before any is added
    constexpr int R = (MT * 2 < 8) ? MT * 2 : 8;   // outputs per thread per pass (pcols <= 512)
    constexpr int QB = 32 / R;                      // slices per batch
    const int n_out = MT * pcols;
    for (int o0 = tid; o0 < n_out; o0 += R * kThreads) {
        float sum[R];
#pragma unroll
        for (int r = 0; r < R; ++r) sum[r] = 0.f;
        for (int q0 = 0; q0 < ks; q0 += QB) {
            float v[R][QB];
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int o = o0 + r * kThreads;
                const int m = o / pcols, col = o - m * pcols;
                const float* src = p.part + pbase + m * kPanelCols + col;
#pragma unroll
                for (int u = 0; u < QB; ++u)
                    v[r][u] = (o < n_out && q0 + u < ks)
                                  ? __hip_atomic_load(src + int64_t(q0 + u) * (MT * kPanelCols), __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT)
                                  : 0.f;
            }
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int u = 0; u < QB; ++u)
                    if (q0 + u < ks) sum[r] += v[r][u];
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int o = o0 + r * kThreads;
            const int m = o / pcols, col = o - m * pcols;
            const int n = chunk0 * 8 + col;
            if (o < n_out && m0 + m < p.M && n < p.N) store_out<CHAIN>(p, b, m0 + m, n, sum[r]);
        }
    }
    if constexpr (CHAIN) signal_done(dep);
}

template <int DT, int MT, int U>
__global__ __launch_bounds__(kThreads) void gemv_kernel(const KParams p) {
    extern __shared__ float lds[];
    __shared__ int s_last;
    gemv_item<DT, MT, U, false>(p, blockIdx.x, lds, &s_last, Dep{});
}

// ---------------------------------------------------------------------------------------------
// The fused decode chain: one persistent launch runs the MatMuls of the chain back to back.
// The work items of all MatMuls form one ordered list (every item of MatMul s precedes every
// item of MatMul s+1); workgroup w takes items w, w + G, w + 2G, ... in that order.  An item of
// MatMul s+1 issues its first W loads at once and only then waits for MatMul s to have
// completed all of its panels, so the next weight stream starts while the previous MatMul's
// last panels are still being gathered -- the paper's point of starting independent work
// earlier, here between consecutive narrow MatMuls.  (A shared claim counter would serialise
// thousands of same-address atomics; the static order costs none.)
//
// Progress: a workgroup finishes all of its items of MatMul s before it waits on MatMul s, and
// it only ever waits on items placed earlier in the list.  So the waits always end once all G
// workgroups are resident; the launch uses at most one workgroup per compute unit so that they
// are, even beside the attention kernel on the other stream.  Every wait is also bounded
// (Dep::spin_limit): if it ever gave up, the error flag is raised instead of the GPU hanging.
// Every workgroup leaves after its last item; the last one out resets the counters.
// ---------------------------------------------------------------------------------------------
constexpr int kChainMax = 5;

struct ChainArgs {
    KParams step[kChainMax];
    int first_item[kChainMax + 1];   // list position of each MatMul's first item
    unsigned panels[kChainMax];      // panels (all batch entries and row blocks) of each MatMul
    unsigned* sync;                  // [1] exited workgroups, [2] error, [3 + s] done of MatMul s
    int n_steps;
    int spin_limit;
    int sleep_reps;
};

__global__ __launch_bounds__(kThreads) void chain_kernel(const ChainArgs a) {
    extern __shared__ float lds[];
    __shared__ int s_last;
    unsigned* sync = a.sync;
    const int total = a.first_item[a.n_steps];
    int st = 0;
    for (int item = blockIdx.x; item < total; item += gridDim.x) {
        while (st + 1 < a.n_steps && item >= a.first_item[st + 1]) ++st;
        Dep dep;
        dep.wait_on = st ? sync + 3 + (st - 1) : nullptr;
        dep.target = st ? a.panels[st - 1] : 0;
        dep.done = sync + 3 + st;
        dep.error = sync + 2;
        dep.spin_limit = a.spin_limit;
        dep.sleep_reps = a.sleep_reps;
        gemv_item<NMM_BF16, 1, 4, true>(a.step[st], item - a.first_item[st], lds, &s_last, dep);
        __syncthreads();   // LDS is reused by the next item
    }
    // leave: the last workgroup out resets the completion counters for the next launch
    if (threadIdx.x == 0) {
        __builtin_amdgcn_s_waitcnt(0);
        const unsigned prev = __hip_atomic_fetch_add(sync + 1, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (prev == gridDim.x - 1) {
            for (int i = 0; i < a.n_steps; ++i)
                __hip_atomic_store(sync + 3 + i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(sync + 1, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// y = 0 (and its bf16 copy) for K == 0: the empty sum.
__global__ void zero_output_kernel(float* y, int64_t ldy, int64_t sy, uint16_t* ybf, int64_t group,
                                   int64_t keep, int64_t ldm, int64_t sb, int64_t M, int64_t N,
                                   int64_t batch) {
    const int64_t total = batch * M * N;
    for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < total;
         i += int64_t(gridDim.x) * blockDim.x) {
        const int64_t n = i % N, m = (i / N) % M, b = i / (N * M);
        y[b * sy + m * ldy + n] = 0.f;
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
    hipLaunchKernelGGL((gemv_kernel<DT, MT, U>), dim3(static_cast<uint32_t>(grid)), dim3(kThreads), lds, s, kp);
}

template <int DT, int MT>
void launch_u(const KParams& kp, int64_t grid, size_t lds, int unroll, hipStream_t s) {
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

bool chain_fusable(const GemvArgs* a, const GemvPlan* p, int n) {
    if (n < 1 || n > kChainMax) return false;
    for (int i = 0; i < n; ++i)
        if (a[i].dt != NMM_BF16 || a[i].M != 1 || a[i].K == 0 || a[i].N == 0 || a[i].batch == 0 ||
            p[i].mt != 1 || p[i].unroll != 4)
            return false;
    return true;
}

nmm_status launch_chain(const GemvArgs* a, const GemvPlan* p, int n, unsigned* sync, unsigned* const* tickets,
                        float* const* part, int grid, void* stream) {
    ChainArgs ca{};
    ca.n_steps = n;
    ca.sync = sync;
    ca.spin_limit = 1 << 22;   // ~ a second of polling: far beyond any legitimate wait
    ca.sleep_reps = 1;
    if (const char* e = std::getenv("NMM_CHAIN_SLEEP")) ca.sleep_reps = std::max(1, std::atoi(e));
    size_t lds = 0;
    int first = 0;
    for (int i = 0; i < n; ++i) {
        ca.step[i] = make_params(a[i], p[i], tickets[i], part[i]);
        ca.first_item[i] = first;
        first += static_cast<int>(p[i].grid);
        ca.panels[i] = static_cast<unsigned>(a[i].batch * p[i].mblocks * (p[i].n_full + (p[i].tail_chunks ? 1 : 0)));
        lds = std::max(lds, gemv_lds_bytes(p[i]));
    }
    ca.first_item[n] = first;
    grid = std::max(1, std::min(grid, first));
    hipLaunchKernelGGL(chain_kernel, dim3(static_cast<uint32_t>(grid)), dim3(kThreads), lds,
                       static_cast<hipStream_t>(stream), ca);
    return last_launch_status();
}

}  // namespace nmm
