// Work partition of the single-tile kernel: which workgroup owns which input group, gate/up
// unit and down unit (the schedule sets the gate/up deal block and the down phase's
// workgroup count; the defaults are single units and the whole grid).  Shared by the kernel and the host-side schedule checker
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

// Gate/up units are dealt round-robin in blocks of 2^lb consecutive units (lb = 0: single
// units): block b goes to workgroup b mod G, so the j-th unit of workgroup wg is unit
// ((j >> lb) * G + wg) * 2^lb + (j mod 2^lb), and an expert's I/8 units are spread over
// about (I/8) / 2^lb workgroups.  The last block of the phase may be partial.
__host__ __device__ __forceinline__ int up_count(int wg, int G, int n_up, int lb) {
    const int nb = (n_up + (1 << lb) - 1) >> lb;   // blocks
    if (nb <= wg) return 0;
    const int mine = (nb - 1 - wg) / G + 1;         // blocks of this workgroup
    const int cut = ((nb - 1) % G == wg) ? (nb << lb) - n_up : 0;   // missing tail of the last block
    return (mine << lb) - cut;
}
__host__ __device__ __forceinline__ int up_unit(int wg, int G, int j, int lb) {
    return (((j >> lb) * G + wg) << lb) | (j & ((1 << lb) - 1));
}

// Contiguous ranges (down units, exchanged input groups): items [range_lo(wg), range_lo(wg + 1))
// of n go to workgroup wg (n * G < 2^32).
__host__ __device__ __forceinline__ int range_lo(int wg, int G, int n) {
    return (int)((uint32_t)wg * (uint32_t)n / (uint32_t)G);
}

// Down units go in contiguous ranges to the first Gd workgroups of the grid (Gd <= G; the
// others have none): [down_lo(wg), down_lo(wg + 1)).
__host__ __device__ __forceinline__ int down_lo(int wg, int Gd, int n_dn) {
    return wg < Gd ? range_lo(wg, Gd, n_dn) : n_dn;
}

}  // namespace monomoe
