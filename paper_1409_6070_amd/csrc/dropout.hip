// Dropout per level (Section 2.1): one rate for the input of every convolution
// that is not 1x1 (Section 2.2 applies none to the network-in-network layers)
// and one for the softmax layer's input.  Inverted dropout on rows >= 1 of a
// feature matrix; the ground row is copied unchanged, so every inactive site
// keeps the layer's shared ground state.  The masks are recomputed from the
// counter-based generator wherever they are needed (here and in the backward
// epilogues), never stored.

#include "common.h"
#include "kernels.h"

namespace sscn {

// Xd = X with rows 1 .. n multiplied by their dropout factors (16 bytes per
// thread: VE consecutive channels of one row, VE / 4 generator calls).  Rows
// first .. n: first = 0 copies the ground row; first = 1 works in place (X ==
// Xd, each element read and written by one thread), as the backward pass does
// on the gradient below a dropout level.
template <typename T>
__global__ void __launch_bounds__(256) k_dropout_rows(const T* X, T* Xd, int32_t cp, const int32_t* __restrict__ n_rows,
                                                      int32_t first, DropArgs d) {
  constexpr int VE = Elem<T>::VE;
  const int vpr = cp / VE;
  const int64_t total = (int64_t)(*n_rows + 1 - first) * vpr;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = first + t / vpr;
    const int v = (int)(t - (r - first) * vpr);
    Vec16 x = ((const Vec16*)(X + r * cp))[v];
    if (r >= 1) {
      const uint32_t q = (uint32_t)d.keys[r - 1];
#pragma unroll
      for (int h = 0; h < VE / 4; ++h) {
        float f[4];
        drop_factors4(d, q, (uint32_t)(v * (VE / 4) + h), f);
#pragma unroll
        for (int e = 0; e < 4; ++e) ((T*)&x)[h * 4 + e] = Elem<T>::from_f32(Elem<T>::to_f32(((T*)&x)[h * 4 + e]) * f[e]);
      }
    }
    ((Vec16*)(Xd + r * cp))[v] = x;
  }
}

// The softmax layer's input with dropout: hd[b] = X_top[head_rows[b]] times the
// factors of row key b (every sample, the empty ones -- ground row -- included).
template <typename T>
__global__ void __launch_bounds__(256) k_head_drop(const T* __restrict__ X_top, const int32_t* __restrict__ head_rows,
                                                   int32_t batch, int32_t cp, T* __restrict__ hd, DropArgs d) {
  constexpr int VE = Elem<T>::VE;
  const int vpr = cp / VE;
  const int64_t total = (int64_t)batch * vpr;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += (int64_t)gridDim.x * blockDim.x) {
    const int b = (int)(t / vpr);
    const int v = (int)(t - (int64_t)b * vpr);
    Vec16 x = ((const Vec16*)(X_top + (int64_t)head_rows[b] * cp))[v];
#pragma unroll
    for (int h = 0; h < VE / 4; ++h) {
      float f[4];
      drop_factors4(d, (uint32_t)b, (uint32_t)(v * (VE / 4) + h), f);
#pragma unroll
      for (int e = 0; e < 4; ++e) ((T*)&x)[h * 4 + e] = Elem<T>::from_f32(Elem<T>::to_f32(((T*)&x)[h * 4 + e]) * f[e]);
    }
    ((Vec16*)(hd + (int64_t)b * cp))[v] = x;
  }
}

static int drop_grid(int64_t items) {
  return (int)std::max<int64_t>(1, std::min<int64_t>((items + 255) / 256, 2048));
}

hipError_t launch_dropout_rows(bool bf16, const void* X, void* Xd, int32_t cp, const int32_t* n_rows, int64_t max_rows,
                               const DropArgs& d, hipStream_t st) {
  const int grid = drop_grid(max_rows * (cp / (bf16 ? 8 : 4)));
  const int32_t first = X == Xd ? 1 : 0;
  if (bf16)
    hipLaunchKernelGGL(k_dropout_rows<__bf16>, dim3(grid), dim3(256), 0, st, (const __bf16*)X, (__bf16*)Xd, cp, n_rows,
                       first, d);
  else
    hipLaunchKernelGGL(k_dropout_rows<float>, dim3(grid), dim3(256), 0, st, (const float*)X, (float*)Xd, cp, n_rows,
                       first, d);
  return hipGetLastError();
}

hipError_t launch_head_drop(bool bf16, const void* X_top, const int32_t* head_rows, int32_t batch, int32_t cp,
                            void* hd, const DropArgs& d, hipStream_t st) {
  if (batch <= 0) return hipSuccess;
  const int grid = drop_grid((int64_t)batch * (cp / (bf16 ? 8 : 4)));
  if (bf16)
    hipLaunchKernelGGL(k_head_drop<__bf16>, dim3(grid), dim3(256), 0, st, (const __bf16*)X_top, head_rows, batch, cp,
                       (__bf16*)hd, d);
  else
    hipLaunchKernelGGL(k_head_drop<float>, dim3(grid), dim3(256), 0, st, (const float*)X_top, head_rows, batch, cp,
                       (float*)hd, d);
  return hipGetLastError();
}

}  // namespace sscn
