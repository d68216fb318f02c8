// Work partition of the single-tile kernel: which workgroup owns which input group, gate/up
// unit and down unit.  Shared by the kernel and the host-side schedule checker
// (monomoe_schedule.hip), so that both use the same arithmetic.  Router rows (expert e on
// workgroup e mod G) and output chunks (chunk r on workgroup r mod G, wavefront
// (r / G) mod kWaves) are dealt round-robin by the kernels' loops.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace monomoe {

// A small input (at most this many 8-element chunks per thread of a workgroup) is quantised
// by every workgroup into its own LDS; a larger one is quantised once, split over the
// workgroups, and exchanged.
constexpr int kLocalQuantChunks = 16;

// Gate/up units are dealt round-robin: the j-th of workgroup wg's units is unit wg + G*j.
__host__ __device__ __forceinline__ int up_count(int wg, int G, int n_up) {
    return n_up > wg ? (n_up - 1 - wg) / G + 1 : 0;
}
__host__ __device__ __forceinline__ int up_unit(int wg, int G, int j) { return wg + G * j; }

// Contiguous ranges (down units, exchanged input groups): items [range_lo(wg), range_lo(wg + 1))
// of n go to workgroup wg (n * G < 2^32).
__host__ __device__ __forceinline__ int range_lo(int wg, int G, int n) {
    return (int)((uint32_t)wg * (uint32_t)n / (uint32_t)G);
}

}  // namespace monomoe
