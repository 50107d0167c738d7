// One stochastic-gradient-descent update of every parameter array (training by
// backpropagation, Section 3): classical momentum with L2 weight decay,
//   v = momentum * v + (g + wd * w),  w = w - lr * v,
// on float32 master weights, then the storage-dtype copy the next forward pass
// reads.  All arrays of a step in one launch: blockIdx selects an array (by
// the block ranges in blk_beg) and a span of it; memory-bound, one element per
// thread and coalesced.

#include "common.h"
#include "kernels.h"

namespace sscn {

static_assert(sizeof(SgdArgs) <= 4096, "kernel arguments must fit the 4 KiB argument segment");

__global__ void __launch_bounds__(256) k_sgd(SgdArgs a) {
  int j = 0;
  while (j + 1 < a.njobs && (int)blockIdx.x >= a.blk_beg[j + 1]) ++j;
  const SgdJob& J = a.job[j];
  const int64_t nblk = a.blk_beg[j + 1] - a.blk_beg[j];
  for (int64_t i = (int64_t)(blockIdx.x - a.blk_beg[j]) * blockDim.x + threadIdx.x; i < J.n;
       i += nblk * blockDim.x) {
    const float w = J.w[i];
    const float v = a.momentum * J.v[i] + (J.g[i] + J.wd * w);
    const float wn = w - a.lr * v;
    J.v[i] = v;
    J.w[i] = wn;
    if (J.w_store) {
      if (a.store_bf16)
        ((__bf16*)J.w_store)[i] = Elem<__bf16>::from_f32(wn);
      else
        ((float*)J.w_store)[i] = wn;
    }
  }
}

hipError_t launch_sgd(const SgdArgs& a, hipStream_t st) {
  if (a.njobs <= 0 || a.blk_beg[a.njobs] <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_sgd, dim3(a.blk_beg[a.njobs]), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace sscn
