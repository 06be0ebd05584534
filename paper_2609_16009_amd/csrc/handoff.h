// The hand-off between the workgroups of one launch that each produce part of a result and the
// one that combines them: the split-K gather (Algorithm 1's wait for all vector units before the
// accumulate, Section III-B) and the count of finished panels before the cache entry.
//
// Ordering argument (gfx950 ISA), in place of a release/acquire pair:
//  * every value handed over is written with device-scope atomic stores (the SC1 scope bits),
//    which write through the XCD's L2 to the device's coherence point, and read with
//    device-scope atomic loads, which are served from that point, never from a stale L2 line;
//  * a workgroup counts its part in only after `s_waitcnt 0` in every wave and a barrier:
//    a store's counter is decremented when the coherence point acknowledges it, so all of the
//    part's stores are visible there before the count is issued;
//  * the count is a device-scope atomic performed at the coherence point, and the combining
//    workgroup issues its loads only after the count has returned (its value decides whether
//    they run at all), so they reach the coherence point after every part's stores.
// A release/acquire pair at agent scope would add an L2 write-back (buffer_wbl2) to every
// part and an L2 invalidate to the last: measured at +6 us on the [16384, 7168] launch (40.4 to
// 46.3 us) and +0.8 us on [7168, 2112], for no ordering the sequence above lacks.
#pragma once
#include <hip/hip_runtime.h>

namespace nmm {

// Called by one thread of a workgroup after every thread's device-scope stores of its part have
// completed (s_waitcnt 0 in each wave) and the workgroup has met at a barrier.  Counts the part
// in at `counter` and returns whether it was the last of `parts`; the last resets the counter
// to zero for the next launch.
__device__ __forceinline__ bool arrive(unsigned* counter, unsigned parts) {
    const unsigned prev = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (prev != parts - 1) return false;
    __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return true;
}

}  // namespace nmm
