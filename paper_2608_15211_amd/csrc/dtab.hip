// dtab.hip - the last step of the bias-table gradient (Sec. IV-A: the
// relative-position bias of the Swin blocks is a learned table, so its
// gradient is the sum of dS over every pair that reads each entry).
//
// The attention backward kernels leave one partial table per (head, slice)
// of their persistent grid; this kernel sums the slices of each entry in
// slice order, so the result is the same bit for bit on every run.
#include "terra_common.h"

namespace terra {

constexpr int kReduceThreads = 256;

// dT[bin][h] = sum over slices of partial[h][slice][bin].  Consecutive
// threads take consecutive bins of one head, so each slice's loads are
// contiguous, and the loop is unrolled so that loads issue ahead of the
// additions, which stay in slice order.
__global__ __launch_bounds__(kReduceThreads) void dtab_reduce_kernel(
    const float* __restrict__ partial, float* __restrict__ dtab, Geo g, int nslice) {
  const int idx = blockIdx.x * kReduceThreads + threadIdx.x;
  if (idx >= g.nbins * g.heads) return;
  const int h = idx / g.nbins;
  const int bin = idx - h * g.nbins;
  const float* p = partial + (int64_t)h * nslice * g.nbins + bin;
  float acc = 0.0f;
#pragma unroll 8
  for (int s = 0; s < nslice; ++s) acc += p[(int64_t)s * g.nbins];
  dtab[bin * g.heads + h] = acc;
}

// partial: heads x nslice x nbins floats (device); dtab: nbins x heads.
hipError_t launch_dtab_reduce(const Geo& g, const float* partial, float* dtab, int nslice,
                              hipStream_t st) {
  const int nred = g.nbins * g.heads;
  hipLaunchKernelGGL(dtab_reduce_kernel, dim3((nred + kReduceThreads - 1) / kReduceThreads),
                     dim3(kReduceThreads), 0, st, partial, dtab, g, nslice);
  return hipGetLastError();
}

}  // namespace terra
