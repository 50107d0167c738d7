// Epilogue of the gather GEMMs: bias, rectifier, the rectifier derivative of
// the layer below, storage rounding.
#pragma once

#include "common.h"
#include "kernels.h"

namespace sscn {

template <typename T>
__device__ inline float epi_value(const GemmArgs& a, float v, float bias) {
  v += bias;
  if (a.epi == EPI_BIAS_RELU) v = fmaxf(v, 0.f);
  if (a.epi == EPI_BIAS_LRELU) v = v >= 0.f ? v : v / 3.f;
  return v;
}

// Epilogues that store in the storage dtype (the others store float32).
__device__ inline bool epi_stores_T(int epi) {
  return epi == EPI_BIAS_RELU || epi == EPI_STORE || epi == EPI_BIAS_LRELU || epi == EPI_STORE_MASK;
}

template <typename T>
__device__ inline void store_out(const GemmArgs& a, int64_t m, int n, float v) {
  const int64_t o = m * a.out_stride + n;
  if (a.epi == EPI_STORE_MASK)
    v *= act_factor(Elem<T>::to_f32(((const T*)a.mask)[m * a.mask_stride + n]), a.slope);
  if (epi_stores_T(a.epi))
    ((T*)a.out)[o] = Elem<T>::from_f32(v);
  else
    ((float*)a.out)[o] = v;
}

}  // namespace sscn
