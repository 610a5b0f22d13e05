// Workgroup scan used by the accept/reject and drafter sampling kernels.
#pragma once

#include "device_util.h"

namespace dsi {

// inclusive scan of one double per thread over a workgroup of NW waves, with a
// fixed association (wave scan, then the wave totals in order); sh holds NW
// doubles.  Every thread of the workgroup must call it.
template <int NW>
__device__ __forceinline__ double block_scan_incl(double v, double* sh) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double t = __shfl_up(v, o);
    if (lane >= o) v += t;
  }
  if (lane == 63) sh[w] = v;
  __syncthreads();
  double off = 0.0;
  for (int i = 0; i < w; ++i) off += sh[i];
  __syncthreads();
  return off + v;
}

}  // namespace dsi
