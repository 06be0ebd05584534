// Narrow MatMul on the matrix cores for larger M (gfx950): y[M,N] = x[M,K] . W[K,N] with M in
// tiles of 16 or 32 rows, W row-major [K,N] (bf16 or fp16), fp32 accumulation.
//
// Once x has enough rows the streaming GEMV runs out of vector ALU (it spends 2*M flops per
// weight element against HBM's ~1 byte per element), while the product stays HBM-bound for
// the matrix cores far beyond M = 32.  The paper's narrow-dimension conditions (Condition 2,
// Section III-A; Conditions 4-5, Section V) are about where the split between the two units
// lies; on MI355X it is measured, and nmm_gemv's AUTO path switches here above it.
//
//  * A workgroup (4 waves) owns one 128-column panel of W and one K-slice.
//  * W streams in stages of 64 rows x 128 columns (16 KB) together with the stage's 64 k of the
//    x tile (the MFMA A operand, 2-4 KB): each thread keeps two stages of 16-byte chunks in
//    flight, stores the oldest to a double-buffered LDS stage and reloads its registers in
//    place.  The waves read their v_mfma_f32_16x16x32 B operands back with ds_read_b64_tr_b16,
//    the gfx950 transposing LDS read (the B operand needs 8 consecutive k of one column; W rows
//    hold consecutive columns).  x travels with W instead of being staged for the whole slice
//    up front, so no workgroup waits for its x before its W stream starts and the slice length
//    is not bounded by LDS.
//  * Wave w owns the column tiles 2w and 2w+1 of the panel, so no cross-wave reduction is needed.
//  * K-slices are combined exactly like the GEMV's: device-scope atomic partial stores, a
//    ticket per panel, and the last workgroup sums the slices in order.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "bf16_cast.h"
#include "handoff.h"
#include "nmm_internal.h"

namespace nmm {
namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __fp16 fp16x4 __attribute__((__vector_size__(4 * sizeof(__fp16))));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) fp16x4 lds_f16x4;

constexpr int kRsrcWord3 = 0x00020000;
constexpr int kLoadNT = 2;
constexpr uint32_t kOutOfRange = 0x80000000u;
constexpr int kWStride = kMfmaPanelCols + 8;   // LDS row stride of a W stage (elements)
constexpr int kXStride = kMfmaStageRows + 8;   // LDS row stride of an x stage (elements)
constexpr int kMfmaDepth = 2;                  // stages in flight per thread (2-4 measured alike)

struct MParams {
    const uint16_t* x;
    int64_t ldx;
    const uint16_t* w;
    float* y;              // fp32 output (may be null when ybf is set)
    int64_t ldy;
    uint16_t* ybf;         // optional bf16 output, ybf[m * ldyb + n]
    int64_t ldyb;
    int away;              // bf16 rounding: 0 nearest-even, 1 ties away from zero
    float* part;
    unsigned* tickets;
    int M, K, N;
    uint32_t row_bytes, w_extent;
    int panels, ks, rows, items, mblocks;
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kRsrcWord3);
}

// An output: fp32 y only (BF false), or the bf16 copy and, when y is not null, y as well.
template <bool BF>
__device__ __forceinline__ void put_y(const MParams& p, int m, int n, float v) {
    if constexpr (BF) {
        if (p.y) p.y[int64_t(m) * p.ldy + n] = v;
        p.ybf[int64_t(m) * p.ldyb + n] = to_bf16_mode(v, p.away);
    } else {
        p.y[int64_t(m) * p.ldy + n] = v;
    }
}

template <int DT>
__device__ __forceinline__ f32x4 mfma(i32x4 a, i32x4 b, f32x4 c) {
    if constexpr (DT == NMM_BF16)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// B operand of one 16-column tile for 32 k-rows starting at `row0` of the LDS stage: lane
// (g = lane/16, j = lane%16) receives W[row0 + 8g .. + 7][col0 + j] via two transposing reads.
template <int DT>
__device__ __forceinline__ i32x4 load_b(const uint16_t* wst, int row0, int col0, int g, int j) {
    const uint16_t* base = wst + (row0 + 8 * g + (j >> 2)) * kWStride + col0 + 4 * (j & 3);
    uint2 lo, hi;
    if constexpr (DT == NMM_BF16) {
        lo = __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(base)));
        hi = __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(base + 4 * kWStride)));
    } else {
        lo = __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4f16((lds_f16x4*)(base)));
        hi = __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4f16((lds_f16x4*)(base + 4 * kWStride)));
    }
    return i32x4{int(lo.x), int(lo.y), int(hi.x), int(hi.y)};
}

template <int DT, int MT, int D, bool BF>
__global__ __launch_bounds__(kThreads) void mfma_gemv_kernel(const MParams p) {
    // two stage buffers, each a W tile [64][kWStride] followed by an x tile [MT][kXStride]
    extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
    __shared__ int s_last;
    constexpr int MTILES = MT / 16;
    constexpr int kStage = kMfmaStageRows * kWStride + MT * kXStride;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, j = lane & 15;

    const uint32_t bid = blockIdx.x;
    const int item = static_cast<int>(bid % uint32_t(p.items));
    const int mb = static_cast<int>(bid / uint32_t(p.items));
    const int panel = item / p.ks, slice = item - panel * p.ks;
    const int m0 = mb * MT, k0 = slice * p.rows, n0 = panel * kMfmaPanelCols;
    const int stages = (min(p.rows, p.K - k0) + kMfmaStageRows - 1) / kMfmaStageRows;
    const int mrows = min(MT, p.M - m0);

    // ---- W: thread t takes chunk t%16 of rows t/16 + 16q (q < 4) of a stage.
    const __amdgpu_buffer_rsrc_t wr = make_rsrc(p.w, p.w_extent);
    const int wc = tid & 15, wr0 = tid >> 4;
    const int chunks_valid = min(16, (p.N - n0 + 7) / 8);
    auto w_off = [&](int st, int q) -> uint32_t {
        const int row = k0 + st * kMfmaStageRows + wr0 + 16 * q;
        return (st < stages && row < p.K && wc < chunks_valid) ? uint32_t(row) * p.row_bytes + uint32_t(n0 / 8 + wc) * 16u
                                                              : kOutOfRange;
    };
    // ---- x: thread t takes chunk t%8 (8 k) of row t/8 of the stage's 64 k; rows past M or
    // chunks past K read zeros, and elements past K inside the last chunk are cleared on the way
    // to LDS (the padding of a row is read but never used).
    const int xm = tid >> 3, xc = tid & 7;
    const __amdgpu_buffer_rsrc_t xr =
        make_rsrc(p.x + int64_t(m0) * p.ldx, uint32_t(((mrows - 1) * p.ldx + (p.K + 7) / 8 * 8) * 2));
    const int xk_left = p.K - (k0 + 8 * xc);   // elements of this thread's chunk of stage 0 inside K
    auto x_off = [&](int st) -> uint32_t {
        const int left = xk_left - st * kMfmaStageRows;
        return (st < stages && xm < mrows && left > 0) ? uint32_t((xm * p.ldx + k0 + st * kMfmaStageRows + 8 * xc) * 2)
                                                      : kOutOfRange;
    };

    // D stages in flight: the registers of stage s go to LDS and are then reloaded with stage
    // s + D in place (no register copies, so the stream never drains); past the slice they read
    // zeros without touching memory.
    i32x4 wreg[D][4], xreg[D];
#pragma unroll
    for (int d = 0; d < D; ++d) {
#pragma unroll
        for (int q = 0; q < 4; ++q) wreg[d][q] = __builtin_amdgcn_raw_buffer_load_b128(wr, w_off(d, q), 0, kLoadNT);
        xreg[d] = __builtin_amdgcn_raw_buffer_load_b128(xr, x_off(d), 0, 0);
    }

    f32x4 acc[MTILES][2];
#pragma unroll
    for (int mt = 0; mt < MTILES; ++mt)
#pragma unroll
        for (int t = 0; t < 2; ++t) acc[mt][t] = f32x4{0.f, 0.f, 0.f, 0.f};

    // one stage: registers to LDS buffer (s & 1), reload with stage s + D, then the MFMAs.  A
    // wave that writes buffer (s & 1) has passed the barrier of stage s - 1, so every wave has
    // finished reading stage s - 2 from it.
    auto stage = [&](int s, i32x4 (&wd)[4], i32x4& xd) {
        uint16_t* wst = smem + (s & 1) * kStage;
        uint16_t* xst = wst + kMfmaStageRows * kWStride;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            *reinterpret_cast<i32x4*>(wst + (wr0 + 16 * q) * kWStride + 8 * wc) = wd[q];
            wd[q] = __builtin_amdgcn_raw_buffer_load_b128(wr, w_off(s + D, q), 0, kLoadNT);
        }
        if (tid < MT * 8) {
            i32x4 v = xd;
            if (p.K & 7) {
                const int left = xk_left - s * kMfmaStageRows;
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] &= (2 * e + 1 < left) ? -1 : (2 * e < left ? 0x0000FFFF : 0);
            }
            *reinterpret_cast<i32x4*>(xst + xm * kXStride + 8 * xc) = v;
        }
        xd = __builtin_amdgcn_raw_buffer_load_b128(xr, x_off(s + D), 0, 0);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < kMfmaStageRows / 32; ++kk) {
            i32x4 a[MTILES];
#pragma unroll
            for (int mt = 0; mt < MTILES; ++mt)
                a[mt] = *reinterpret_cast<const i32x4*>(xst + (16 * mt + j) * kXStride + 32 * kk + 8 * g);
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const i32x4 b = load_b<DT>(wst, 32 * kk, 16 * (2 * wave + t), g, j);
#pragma unroll
                for (int mt = 0; mt < MTILES; ++mt) acc[mt][t] = mfma<DT>(a[mt], b, acc[mt][t]);
            }
        }
    };
    int s0 = 0;
    for (; s0 + D <= stages; s0 += D) {
#pragma unroll
        for (int d = 0; d < D; ++d) stage(s0 + d, wreg[d], xreg[d]);
    }
#pragma unroll
    for (int d = 0; d + 1 < D; ++d)
        if (s0 + d < stages) stage(s0 + d, wreg[d], xreg[d]);

    // ---- outputs: lane (g, j) holds rows 4g+i of its tiles, column j
    const int64_t pbase = ((int64_t(mb) * p.panels + panel) * p.ks) * (int64_t(MT) * kMfmaPanelCols);
    if (p.ks == 1) {
#pragma unroll
        for (int mt = 0; mt < MTILES; ++mt)
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int m = m0 + 16 * mt + 4 * g + i, n = n0 + 16 * (2 * wave + t) + j;
                    if (m < p.M && n < p.N) put_y<BF>(p, m, n, acc[mt][t][i]);
                }
        return;
    }
#pragma unroll
    for (int mt = 0; mt < MTILES; ++mt)
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = 16 * mt + 4 * g + i, c = 16 * (2 * wave + t) + j;
                __hip_atomic_store(p.part + pbase + int64_t(slice) * (MT * kMfmaPanelCols) + r * kMfmaPanelCols + c,
                                   acc[mt][t][i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
    // same hand-off as the GEMV: completed device-scope stores, one ticket, ordered gather
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) {
        s_last = arrive(p.tickets + int64_t(mb) * p.panels + panel, unsigned(p.ks));
    }
    __syncthreads();
    if (!s_last) return;
    // every output of the panel sums its slices in slice order; the loads of PER outputs x QB
    // slices are all in flight before any is added
    constexpr int PER = MT * kMfmaPanelCols / kThreads;   // outputs per thread (8 or 16)
    constexpr int QB = 64 / PER;                            // slices per batch
    float sum[PER];
#pragma unroll
    for (int r = 0; r < PER; ++r) sum[r] = 0.f;
    for (int q0 = 0; q0 < p.ks; q0 += QB) {
        float v[PER][QB];
#pragma unroll
        for (int r = 0; r < PER; ++r)
#pragma unroll
            for (int u = 0; u < QB; ++u) {
                const int o = tid + r * kThreads;
                v[r][u] = (q0 + u < p.ks)
                              ? __hip_atomic_load(p.part + pbase + int64_t(q0 + u) * (MT * kMfmaPanelCols) + o,
                                                  __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                              : 0.f;
            }
#pragma unroll
        for (int r = 0; r < PER; ++r)
#pragma unroll
            for (int u = 0; u < QB; ++u)
                if (q0 + u < p.ks) sum[r] += v[r][u];
    }
#pragma unroll
    for (int r = 0; r < PER; ++r) {
        const int o = tid + r * kThreads;
        const int m = m0 + o / kMfmaPanelCols, n = n0 + o % kMfmaPanelCols;
        if (m < p.M && n < p.N) put_y<BF>(p, m, n, sum[r]);
    }
}

template <int DT, int MT>
void launch_mt(const MParams& mp, int64_t grid, size_t lds, hipStream_t s) {
    if (mp.ybf)
        hipLaunchKernelGGL((mfma_gemv_kernel<DT, MT, kMfmaDepth, true>), dim3(static_cast<uint32_t>(grid)), dim3(kThreads), lds, s, mp);
    else
        hipLaunchKernelGGL((mfma_gemv_kernel<DT, MT, kMfmaDepth, false>), dim3(static_cast<uint32_t>(grid)), dim3(kThreads), lds, s, mp);
}

}  // namespace

size_t mfma_lds_bytes(const GemvPlan& p) {
    return size_t(2) * (kMfmaStageRows * kWStride + p.mt * kXStride) * 2;
}

nmm_status launch_mfma(const GemvArgs& a, const GemvPlan& p, unsigned* tickets, float* part, void* stream) {
    MParams mp{};
    mp.x = static_cast<const uint16_t*>(a.x);
    mp.ldx = a.ldx;
    mp.w = static_cast<const uint16_t*>(a.w);
    mp.y = a.y;
    mp.ldy = a.ldy;
    mp.ybf = static_cast<uint16_t*>(a.ybf);
    mp.ldyb = a.ybf_ldm;
    mp.away = a.ybf_away;
    mp.part = part;
    mp.tickets = tickets;
    mp.M = static_cast<int>(a.M);
    mp.K = static_cast<int>(a.K);
    mp.N = static_cast<int>(a.N);
    mp.row_bytes = static_cast<uint32_t>(a.ldw * 2);
    mp.w_extent = static_cast<uint32_t>(((a.K - 1) * a.ldw + (a.N + 7) / 8 * 8) * 2);
    mp.panels = p.n_full;
    mp.ks = p.ks_full;
    mp.rows = p.rows_full;
    mp.items = p.items;
    mp.mblocks = p.mblocks;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const size_t lds = mfma_lds_bytes(p);
    if (a.dt == NMM_BF16) {
        if (p.mt == 16) launch_mt<NMM_BF16, 16>(mp, p.grid, lds, s);
        else launch_mt<NMM_BF16, 32>(mp, p.grid, lds, s);
    } else {
        if (p.mt == 16) launch_mt<NMM_F16, 16>(mp, p.grid, lds, s);
        else launch_mt<NMM_F16, 32>(mp, p.grid, lds, s);
    }
    return hipGetLastError() == hipSuccess ? NMM_OK : NMM_ERR_HIP;
}

}  // namespace nmm
