// Sparse 2x2 stride-2 max-pooling (Section 2.1) over active sites (Section 2.3).
//
// Forward: output row o takes, channel by channel, the maximum over the four
// rows its window reads (row 0, the ground row, for inactive locations) and
// records the first window position attaining it.  Row 0 passes the ground
// state through.
//
// Backward: windows do not overlap, so each active row below has exactly one
// parent; its gradient is a gather through the parent link (no atomics).  The
// ReLU mask of the convolution below is applied in the same pass, so the
// stored result is dL/dZ of that convolution.  Row 0 (the ground row) sums
// the ground row above and every maximum an active window took from a ground
// location: a two-pass deterministic reduction.

#include "common.h"
#include "kernels.h"

namespace sscn {

template <typename T>
__global__ void __launch_bounds__(256) k_pool_fwd(const T* __restrict__ X_in, int32_t stride_in,
                                                  const int32_t* __restrict__ R, T* X_out, int32_t stride_out,
                                                  uint8_t* argmax, int32_t cp, const int32_t* n_out_p) {
  constexpr int VE = Elem<T>::VE;
  const int nv = cp / VE;
  const int64_t total = (int64_t)(*n_out_p + 1) * nv;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t o = t / nv;
    const int c = (int)(t - o * nv) * VE;
    Vec16 in[4];
#pragma unroll
    for (int f = 0; f < 4; ++f) in[f] = *(const Vec16*)(X_in + (int64_t)R[o * 4 + f] * stride_in + c);
    Vec16 out;
    T* ov = (T*)&out;
    uint8_t am[VE];
#pragma unroll
    for (int j = 0; j < VE; ++j) {
      float best = Elem<T>::to_f32(((const T*)&in[0])[j]);
      int arg = 0;
#pragma unroll
      for (int f = 1; f < 4; ++f) {
        float v = Elem<T>::to_f32(((const T*)&in[f])[j]);
        if (v > best) {
          best = v;
          arg = f;
        }
      }
      ov[j] = ((const T*)&in[arg])[j];
      am[j] = (uint8_t)arg;
    }
    *(Vec16*)(X_out + o * stride_out + c) = out;
    uint8_t* ap = argmax + o * stride_out + c;
#pragma unroll
    for (int j = 0; j < VE; ++j) ap[j] = am[j];
  }
}

template <typename T>
__global__ void __launch_bounds__(256) k_pool_bwd(const T* __restrict__ dY, int32_t stride,
                                                  const uint8_t* __restrict__ argmax, const int32_t* __restrict__ Pt,
                                                  const T* __restrict__ Y_below, T* grad_below, int32_t cp,
                                                  const int32_t* n_in_p) {
  constexpr int VE = Elem<T>::VE;
  const int nv = cp / VE;
  const int64_t total = (int64_t)(*n_in_p) * nv;  // rows 1..n_in
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = 1 + t / nv;
    const int c = (int)(t - (i - 1) * nv) * VE;
    const int p = Pt[i];
    Vec16 y = *(const Vec16*)(Y_below + i * stride + c);
    Vec16 out = {{0u, 0u, 0u, 0u}};
    if (p >= 0) {
      const int64_t o = p >> 2;
      const int f = p & 3;
      Vec16 g = *(const Vec16*)(dY + o * stride + c);
      const uint8_t* ap = argmax + o * stride + c;
#pragma unroll
      for (int j = 0; j < VE; ++j) {
        const bool take = (ap[j] == f) && (Elem<T>::to_f32(((const T*)&y)[j]) > 0.f);
        ((T*)&out)[j] = take ? ((const T*)&g)[j] : Elem<T>::from_f32(0.f);
      }
    }
    *(Vec16*)(grad_below + i * stride + c) = out;
  }
}

// Pass 1: block b sums, per channel, dY[o][c] over its rows o >= 1 whose max came from row 0.
template <typename T>
__global__ void __launch_bounds__(256) k_pool_row0_part(const T* __restrict__ dY, int32_t stride,
                                                        const uint8_t* __restrict__ argmax,
                                                        const int32_t* __restrict__ R, int32_t cp,
                                                        const int32_t* n_out_p, float* part) {
  const int n_out = *n_out_p;
  const int per = (n_out + gridDim.x - 1) / gridDim.x;
  const int o_beg = 1 + blockIdx.x * per;
  const int o_end = min(n_out + 1, o_beg + per);
  for (int c = threadIdx.x; c < cp; c += blockDim.x) {
    float s = 0.f;
    for (int o = o_beg; o < o_end; ++o) {
      const int f = argmax[(int64_t)o * stride + c];
      if (R[(int64_t)o * 4 + f] == 0) s += Elem<T>::to_f32(dY[(int64_t)o * stride + c]);
    }
    part[(int64_t)blockIdx.x * cp + c] = s;
  }
}

// Pass 2: grad_below[0][c] = mask(Y_below[0][c]) * (dY[0][c] + sum of pass-1 partials).
template <typename T>
__global__ void __launch_bounds__(256) k_pool_row0_final(const T* __restrict__ dY, const float* __restrict__ part,
                                                         int32_t nparts, const T* __restrict__ Y_below,
                                                         T* grad_below, int32_t cp) {
  for (int c = blockIdx.x * blockDim.x + threadIdx.x; c < cp; c += gridDim.x * blockDim.x) {
    float s = Elem<T>::to_f32(dY[c]);
    for (int p = 0; p < nparts; ++p) s += part[(int64_t)p * cp + c];
    grad_below[c] = (Elem<T>::to_f32(Y_below[c]) > 0.f) ? Elem<T>::from_f32(s) : Elem<T>::from_f32(0.f);
  }
}

static int grid_for(int64_t items) { return (int)std::max<int64_t>(1, std::min<int64_t>((items + 255) / 256, 4096)); }

hipError_t launch_pool_fwd(bool bf16, const void* X_in, int32_t stride_in, const int32_t* R, void* X_out,
                           int32_t stride_out, uint8_t* argmax, int32_t cp, const int32_t* n_out, int64_t cap_out,
                           hipStream_t st) {
  const int VE = bf16 ? 8 : 4;
  int grid = grid_for((cap_out + 1) * (cp / VE));
  if (bf16)
    hipLaunchKernelGGL(k_pool_fwd<__bf16>, dim3(grid), dim3(256), 0, st, (const __bf16*)X_in, stride_in, R,
                       (__bf16*)X_out, stride_out, argmax, cp, n_out);
  else
    hipLaunchKernelGGL(k_pool_fwd<float>, dim3(grid), dim3(256), 0, st, (const float*)X_in, stride_in, R,
                       (float*)X_out, stride_out, argmax, cp, n_out);
  return hipGetLastError();
}

hipError_t launch_pool_bwd(bool bf16, const void* dY, int32_t stride, const uint8_t* argmax, const int32_t* Pt,
                           const int32_t* R, const void* Y_below, void* grad_below, int32_t cp, const int32_t* n_out,
                           const int32_t* n_in, int64_t cap_in, int64_t cap_out, float* part, int32_t nparts,
                           hipStream_t st) {
  const int VE = bf16 ? 8 : 4;
  int grid = grid_for(cap_in * (cp / VE));
  if (bf16) {
    hipLaunchKernelGGL(k_pool_bwd<__bf16>, dim3(grid), dim3(256), 0, st, (const __bf16*)dY, stride, argmax, Pt,
                       (const __bf16*)Y_below, (__bf16*)grad_below, cp, n_in);
    hipLaunchKernelGGL(k_pool_row0_part<__bf16>, dim3(nparts), dim3(256), 0, st, (const __bf16*)dY, stride, argmax, R,
                       cp, n_out, part);
    hipLaunchKernelGGL(k_pool_row0_final<__bf16>, dim3((cp + 255) / 256), dim3(256), 0, st, (const __bf16*)dY, part,
                       nparts, (const __bf16*)Y_below, (__bf16*)grad_below, cp);
  } else {
    hipLaunchKernelGGL(k_pool_bwd<float>, dim3(grid), dim3(256), 0, st, (const float*)dY, stride, argmax, Pt,
                       (const float*)Y_below, (float*)grad_below, cp, n_in);
    hipLaunchKernelGGL(k_pool_row0_part<float>, dim3(nparts), dim3(256), 0, st, (const float*)dY, stride, argmax, R, cp,
                       n_out, part);
    hipLaunchKernelGGL(k_pool_row0_final<float>, dim3((cp + 255) / 256), dim3(256), 0, st, (const float*)dY, part,
                       nparts, (const float*)Y_below, (float*)grad_below, cp);
  }
  (void)cap_out;
  return hipGetLastError();
}

}  // namespace sscn
