// Mask -> ascending active-neuron index list (rm_mask_compact).
//
// A reference execution's neuron mask is stored as the indices of its selected neurons and shared by every
// step of a denoising group (paper section 4.1, "Group-Shared Neuron Masks"; section 5 builds one mask per
// layer and group).  The kernel turns a uint8 mask into that list.
//
// Grid: one workgroup per (mask, segment of 1024 neurons).  Every workgroup first counts the active neurons of
// its mask before its segment and in total, reading the whole mask (at most a few KB, from L2): the workgroups
// need no communication, so one launch of many small workgroups replaces a serial sweep by one.  It then scans its
// segment (4 neurons per thread: wave inclusive scan, prefix over the four waves) and writes the positions of
// its active neurons, in order, from list slot `before` on; and it fills the slots of its own index range that
// lie past the total with -1.  The list is ascending by construction, and the result is bit-exact and
// independent of scheduling.
#include "rm_units.h"

namespace {

__global__ __launch_bounds__(rm_units::kCompactThreads) void mask_compact_kernel(const uint8_t *__restrict__ mask,
                                                                                 int d_ff, int nseg,
                                                                                 int32_t *__restrict__ idx,
                                                                                 int32_t *__restrict__ count) {
    const int m = blockIdx.x / nseg;
    rm_units::compact_segment(mask, d_ff, m, blockIdx.x - m * nseg, idx, count);
}

}  // namespace

namespace rm {

hipError_t launch_mask_compact(const uint8_t *mask, int n_masks, int d_ff, int32_t *idx, int32_t *count,
                               hipStream_t st) {
    const int nseg = (d_ff + rm_units::kSeg - 1) / rm_units::kSeg;
    hipLaunchKernelGGL(mask_compact_kernel, dim3(nseg * n_masks), dim3(rm_units::kCompactThreads), 0, st, mask, d_ff,
                       nseg, idx, count);
    return hipGetLastError();
}

}  // namespace rm
