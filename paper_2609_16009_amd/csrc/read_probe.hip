// Read-bandwidth calibration: stream a buffer once with the GEMV's load instruction (16-byte,
// non-temporal buffer loads, U in flight per lane, U in {1, 2, 4, 8, 16}) and fold it into one
// checksum per workgroup.
// It measures how fast this GPU can read HBM with that access pattern, the practical ceiling
// the GEMV roofline fractions are compared against.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "nmm_internal.h"

namespace nmm {
namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
constexpr int kRsrcWord3 = 0x00020000;
constexpr int kLoadNT = 2;

template <int U>
__global__ __launch_bounds__(256) void read_probe_kernel(const uint8_t* buf, uint64_t chunks, uint32_t* out) {
    const uint64_t nthreads = uint64_t(gridDim.x) * blockDim.x;
    const uint64_t t = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    uint32_t acc = 0;
    // 1 GiB windows keep buffer offsets 32-bit
    constexpr uint64_t kWin = uint64_t(1) << 26;   // chunks per window (1 GiB)
    for (uint64_t w0 = 0; w0 < chunks; w0 += kWin) {
        const uint64_t wn = (chunks - w0 < kWin) ? chunks - w0 : kWin;
        const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint8_t*>(buf + w0 * 16), (short)0, int(wn * 16), kRsrcWord3);
        // this thread's chunks of the window are t, t + nthreads, ...; U of them stay in flight:
        // a slot is folded in and then reloaded in place (no register copies, no drain)
        const uint64_t n_t = (t < wn) ? (wn - t + nthreads - 1) / nthreads : 0;
        const uint64_t groups = ((wn + nthreads - 1) / nthreads + U - 1) / U;   // the same for every lane
        auto load = [&](uint64_t j) {
            return __builtin_amdgcn_raw_buffer_load_b128(r, j < n_t ? uint32_t((t + j * nthreads) * 16) : 0x80000000u, 0,
                                                         kLoadNT);
        };
        if (groups) {
            i32x4 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) v[u] = load(u);
            for (uint64_t g = 1; g < groups; ++g) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    acc ^= uint32_t(v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3]);
                    v[u] = load(g * U + u);
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) acc ^= uint32_t(v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3]);
        }
    }
    // one word per workgroup, so the loads cannot be dropped
    __shared__ uint32_t red[256];
    red[threadIdx.x] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t x = 0;
        for (int i = 0; i < 256; ++i) x ^= red[i];
        out[blockIdx.x] = x;
    }
}

}  // namespace
}  // namespace nmm

extern "C" nmm_status nmm_read_probe(const void* buf, size_t bytes, uint32_t* out, int64_t grid, int unroll,
                                     void* stream) {
    if (!buf || !out) return NMM_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(buf) & 15u) || bytes % 16) return NMM_ERR_ALIGN;
    if (grid < 1 || grid > (int64_t(1) << 20)) return NMM_ERR_SHAPE;
    const uint64_t chunks = bytes / 16;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const uint8_t* b = static_cast<const uint8_t*>(buf);
    const dim3 g(static_cast<uint32_t>(grid)), blk(256);
    switch (unroll) {
        case 1: hipLaunchKernelGGL(nmm::read_probe_kernel<1>, g, blk, 0, s, b, chunks, out); break;
        case 2: hipLaunchKernelGGL(nmm::read_probe_kernel<2>, g, blk, 0, s, b, chunks, out); break;
        case 4: hipLaunchKernelGGL(nmm::read_probe_kernel<4>, g, blk, 0, s, b, chunks, out); break;
        case 8: hipLaunchKernelGGL(nmm::read_probe_kernel<8>, g, blk, 0, s, b, chunks, out); break;
        case 16: hipLaunchKernelGGL(nmm::read_probe_kernel<16>, g, blk, 0, s, b, chunks, out); break;
        default: return NMM_ERR_ARG;
    }
    return hipGetLastError() == hipSuccess ? NMM_OK : NMM_ERR_HIP;
}
