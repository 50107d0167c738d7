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

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

// Packs VE argmax bytes (VE = 8 or 4) into one integer store/load.
template <int VE>
struct ArgPack;
template <>
struct ArgPack<8> {
  typedef uint64_t W;
};
template <>
struct ArgPack<4> {
  typedef uint32_t W;
};

template <typename T>
__global__ void __launch_bounds__(256) k_pool_fwd(const T* __restrict__ X_in, int32_t stride_in,
                                                  const int32_t* __restrict__ R, T* X_out, int32_t stride_out,
                                                  uint8_t* argmax, int32_t cp, const int32_t* n_out_p) {
  constexpr int VE = Elem<T>::VE;
  typedef typename ArgPack<VE>::W AW;
  const int nv = cp / VE;
  const int64_t total = (int64_t)(*n_out_p + 1) * nv;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t o = t / nv;
    const int c = (int)(t - o * nv) * VE;
    const i32x4 r = *(const i32x4*)(R + o * 4);
    u32x4 in[4];
    in[0] = *(const u32x4*)(X_in + (int64_t)r[0] * stride_in + c);
    in[1] = *(const u32x4*)(X_in + (int64_t)r[1] * stride_in + c);
    in[2] = *(const u32x4*)(X_in + (int64_t)r[2] * stride_in + c);
    in[3] = *(const u32x4*)(X_in + (int64_t)r[3] * stride_in + c);
    u32x4 out;
    T* ov = (T*)&out;
    AW am = 0;
    // every index below is a compile-time constant, so in[] stays in registers;
    // the maximum converts back exactly (bf16 and fp32 values are exact in fp32)
#pragma unroll
    for (int j = 0; j < VE; ++j) {
      float best = Elem<T>::to_f32(((const T*)&in[0])[j]);
      AW arg = 0;
#pragma unroll
      for (int f = 1; f < 4; ++f) {
        const float v = Elem<T>::to_f32(((const T*)&in[f])[j]);
        const bool gt = v > best;
        best = gt ? v : best;
        arg = gt ? (AW)f : arg;
      }
      ov[j] = Elem<T>::from_f32(best);
      am |= arg << (8 * j);
    }
    *(u32x4*)(X_out + o * stride_out + c) = out;
    *(AW*)(argmax + o * stride_out + c) = am;
  }
}

template <typename T>
__global__ void __launch_bounds__(256) k_pool_bwd(const T* __restrict__ dY, int32_t stride,
                                                  const uint8_t* __restrict__ argmax, const int32_t* __restrict__ Pt,
                                                  const T* __restrict__ Y_below, T* grad_below, int32_t cp,
                                                  const int32_t* n_in_p) {
  constexpr int VE = Elem<T>::VE;
  typedef typename ArgPack<VE>::W AW;
  const int nv = cp / VE;
  const int64_t total = (int64_t)(*n_in_p) * nv;  // rows 1..n_in
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = 1 + t / nv;
    const int c = (int)(t - (i - 1) * nv) * VE;
    const int p = Pt[i];
    const u32x4 y = *(const u32x4*)(Y_below + i * stride + c);
    u32x4 out = {0u, 0u, 0u, 0u};
    if (p >= 0) {
      const int64_t o = p >> 2;
      const int f = p & 3;
      const u32x4 g = *(const u32x4*)(dY + o * stride + c);
      const AW am = *(const AW*)(argmax + o * stride + c);
#pragma unroll
      for (int j = 0; j < VE; ++j) {
        const bool take = ((int)((am >> (8 * j)) & 0xff) == f) && (Elem<T>::to_f32(((const T*)&y)[j]) > 0.f);
        ((T*)&out)[j] = take ? ((const T*)&g)[j] : Elem<T>::from_f32(0.f);
      }
    }
    *(u32x4*)(grad_below + i * stride + c) = out;
  }
}

// Ground-row reduction, pass 1.  Block b takes a contiguous range of output
// rows o >= 1; thread t owns channel vector t % nv and every (256/nv)-th row of
// the range, summing dY[o][c] where the max of (o, c) was read from row 0.
// The row lanes are then combined in LDS in a fixed order: deterministic.
template <typename T>
__global__ void __launch_bounds__(256) k_pool_row0_part(const T* __restrict__ dY, int32_t stride,
                                                        const uint8_t* __restrict__ argmax,
                                                        const int32_t* __restrict__ R, int32_t cp,
                                                        const int32_t* n_out_p, float* part) {
  constexpr int VE = Elem<T>::VE;
  typedef typename ArgPack<VE>::W AW;
  __shared__ float red[256 * VE];
  const int nv = cp / VE;
  const int lanes = 256 / nv;  // row lanes (nv <= 256)
  const int t = threadIdx.x;
  const int v = t % nv, rl = t / nv;
  const int n_out = *n_out_p;
  const int per = (n_out + gridDim.x - 1) / gridDim.x;
  const int o_beg = 1 + blockIdx.x * per;
  const int o_end = min(n_out + 1, o_beg + per);
  float acc[VE];
#pragma unroll
  for (int j = 0; j < VE; ++j) acc[j] = 0.f;
  if (rl < lanes) {
    for (int o = o_beg + rl; o < o_end; o += lanes) {
      const i32x4 r = *(const i32x4*)(R + (int64_t)o * 4);
      const AW am = *(const AW*)(argmax + (int64_t)o * stride + v * VE);
      const u32x4 g = *(const u32x4*)(dY + (int64_t)o * stride + v * VE);
#pragma unroll
      for (int j = 0; j < VE; ++j) {
        const int f = (int)((am >> (8 * j)) & 3);
        const int rf = f == 0 ? r.x : (f == 1 ? r.y : (f == 2 ? r.z : r.w));
        if (rf == 0) acc[j] += Elem<T>::to_f32(((const T*)&g)[j]);
      }
    }
  }
#pragma unroll
  for (int j = 0; j < VE; ++j) red[t * VE + j] = acc[j];
  __syncthreads();
  for (int e = t; e < cp; e += 256) {  // channel e = vector e / VE, element e % VE
    const int vv = e / VE, jj = e - vv * VE;
    float s = 0.f;
    for (int l = 0; l < lanes; ++l) s += red[(l * nv + vv) * VE + jj];
    part[(int64_t)blockIdx.x * cp + e] = s;
  }
}

// Pass 2: a block covers 16 channels with 16 groups of 16 threads; group g sums
// partials g, g+16, ...; the 16 group sums are added in a fixed order.
// grad_below[0][c] = mask(Y_below[0][c]) * (dY[0][c] + sum of partials).
template <typename T>
__global__ void __launch_bounds__(256) k_pool_row0_final(const T* __restrict__ dY, const float* __restrict__ part,
                                                         int32_t nparts, const T* __restrict__ Y_below,
                                                         T* grad_below, int32_t cp) {
  __shared__ float red[16][16];
  const int cl = threadIdx.x & 15, grp = threadIdx.x >> 4;
  const int c = blockIdx.x * 16 + cl;
  float s = 0.f;
  if (c < cp)
    for (int p = grp; p < nparts; p += 16) s += part[(int64_t)p * cp + c];
  red[grp][cl] = s;
  __syncthreads();
  if (grp == 0 && c < cp) {
    float tot = 0.f;
    for (int g = 0; g < 16; ++g) tot += red[g][cl];
    tot += Elem<T>::to_f32(dY[c]);
    grad_below[c] = (Elem<T>::to_f32(Y_below[c]) > 0.f) ? Elem<T>::from_f32(tot) : Elem<T>::from_f32(0.f);
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

hipError_t launch_pool_bwd_rows(bool bf16, const void* dY, int32_t stride, const uint8_t* argmax, const int32_t* Pt,
                                const int32_t* R, const void* Y_below, void* grad_below, int32_t cp,
                                const int32_t* n_out, const int32_t* n_in, int64_t cap_in, float* part, int32_t nparts,
                                hipStream_t st) {
  const int VE = bf16 ? 8 : 4;
  int grid = grid_for(cap_in * (cp / VE));
  if (bf16) {
    hipLaunchKernelGGL(k_pool_bwd<__bf16>, dim3(grid), dim3(256), 0, st, (const __bf16*)dY, stride, argmax, Pt,
                       (const __bf16*)Y_below, (__bf16*)grad_below, cp, n_in);
    hipLaunchKernelGGL(k_pool_row0_part<__bf16>, dim3(nparts), dim3(256), 0, st, (const __bf16*)dY, stride, argmax, R,
                       cp, n_out, part);
  } else {
    hipLaunchKernelGGL(k_pool_bwd<float>, dim3(grid), dim3(256), 0, st, (const float*)dY, stride, argmax, Pt,
                       (const float*)Y_below, (float*)grad_below, cp, n_in);
    hipLaunchKernelGGL(k_pool_row0_part<float>, dim3(nparts), dim3(256), 0, st, (const float*)dY, stride, argmax, R, cp,
                       n_out, part);
  }
  return hipGetLastError();
}

hipError_t launch_pool_row0_final(bool bf16, const void* dY, const float* part, int32_t nparts, const void* Y_below,
                                  void* grad_below, int32_t cp, hipStream_t st) {
  if (bf16)
    hipLaunchKernelGGL(k_pool_row0_final<__bf16>, dim3((cp + 15) / 16), dim3(256), 0, st, (const __bf16*)dY, part,
                       nparts, (const __bf16*)Y_below, (__bf16*)grad_below, cp);
  else
    hipLaunchKernelGGL(k_pool_row0_final<float>, dim3((cp + 15) / 16), dim3(256), 0, st, (const float*)dY, part,
                       nparts, (const float*)Y_below, (float*)grad_below, cp);
  return hipGetLastError();
}

}  // namespace sscn
