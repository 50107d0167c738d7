// Input scatter, parameter packing, and the softmax output layer (Section 2.1:
// softmax on the output layer) with its cross-entropy loss.

#include "common.h"
#include "kernels.h"

namespace sscn {

// X0[perm[i]][c] = feats[i][c] (zero padding columns); row 0 = 0, the input ground state.
template <typename T>
__global__ void __launch_bounds__(256) k_scatter_input(const T* __restrict__ feats, int32_t n, int32_t c_in,
                                                       const int32_t* __restrict__ perm, T* X0, int32_t cp0) {
  const int64_t total = (int64_t)(n + 1) * cp0;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = t / cp0;
    const int c = (int)(t - i * cp0);
    if (i == n) {  // the ground row
      X0[c] = Elem<T>::from_f32(0.f);
      continue;
    }
    const int r = perm[i];
    if (r < 1) continue;  // rejected site
    X0[(int64_t)r * cp0 + c] = (c < c_in) ? feats[i * c_in + c] : Elem<T>::from_f32(0.f);
  }
}

template <typename T>
__global__ void __launch_bounds__(256) k_gather_dfeats(const T* __restrict__ grad0, int32_t cp0,
                                                       const int32_t* __restrict__ perm, int32_t n, int32_t c_in,
                                                       T* dfeats) {
  const int64_t total = (int64_t)n * c_in;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = t / c_in;
    const int c = (int)(t - i * c_in);
    const int r = perm[i];
    dfeats[t] = (r >= 1) ? grad0[(int64_t)r * cp0 + c] : Elem<T>::from_f32(0.f);
  }
}

template <typename T>
__global__ void __launch_bounds__(256) k_pack(int mode, const T* __restrict__ W, int32_t A, int32_t c_in,
                                              int32_t c_out, int32_t cp_in, int32_t cp_out, T* Bt, int32_t Npad,
                                              int32_t Kpad) {
  const int64_t total = (int64_t)Npad * Kpad;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += (int64_t)gridDim.x * blockDim.x) {
    const int n = (int)(t / Kpad), k = (int)(t - (int64_t)n * Kpad);
    T v = Elem<T>::from_f32(0.f);
    if (mode == 0) {  // Bt[n = out channel][k = f*cp_in + c]
      const int f = k / cp_in, c = k - f * cp_in;
      if (n < c_out && f < A && c < c_in) v = W[((int64_t)f * c_in + c) * c_out + n];
    } else {  // Bt[n = in channel c][k = f*cp_out + o]
      const int f = k / cp_out, o = k - f * cp_out;
      if (n < c_in && f < A && o < c_out) v = W[((int64_t)f * c_in + n) * c_out + o];
    }
    Bt[t] = v;
  }
}

// One workgroup per sample: softmax over the logits, the sample's loss term and
// dL/dlogits = (softmax - onehot) / batch.
template <typename T>
__global__ void __launch_bounds__(256) k_softmax_xent(const float* __restrict__ logits,
                                                      const int32_t* __restrict__ labels, int32_t batch,
                                                      int32_t classes, T* dlogits, int32_t dl_stride,
                                                      float* loss_part) {
  __shared__ float red[256];
  const int b = blockIdx.x;
  const float* z = logits + (int64_t)b * classes;
  float mx = -INFINITY;
  for (int c = threadIdx.x; c < classes; c += blockDim.x) mx = fmaxf(mx, z[c]);
  red[threadIdx.x] = mx;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (threadIdx.x < off) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + off]);
    __syncthreads();
  }
  mx = red[0];
  __syncthreads();
  float s = 0.f;
  for (int c = threadIdx.x; c < classes; c += blockDim.x) s += expf(z[c] - mx);
  red[threadIdx.x] = s;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (threadIdx.x < off) red[threadIdx.x] += red[threadIdx.x + off];
    __syncthreads();
  }
  const float sum = red[0];
  const int label = labels[b];
  const float inv_b = 1.f / (float)batch;
  for (int c = threadIdx.x; c < dl_stride; c += blockDim.x) {
    float g = 0.f;
    if (c < classes) g = (expf(z[c] - mx) / sum - (c == label ? 1.f : 0.f)) * inv_b;
    dlogits[(int64_t)b * dl_stride + c] = Elem<T>::from_f32(g);
  }
  if (threadIdx.x == 0) {
    const bool ok = label >= 0 && label < classes;
    loss_part[b] = ok ? (logf(sum) + mx - z[label]) : 0.f;
  }
}

__global__ void k_loss_final(const float* __restrict__ loss_part, int32_t batch, float* loss) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    float s = 0.f;
    for (int b = 0; b < batch; ++b) s += loss_part[b];
    *loss = batch > 0 ? s / (float)batch : 0.f;
  }
}

// grad_top[row(b)] = mask * dh[b] for non-empty samples; grad_top[0] = mask0 * sum of dh over empty samples.
template <typename T>
__global__ void __launch_bounds__(256) k_head_scatter(const float* __restrict__ dh, int32_t dh_stride,
                                                      const int32_t* __restrict__ head_rows, int32_t batch,
                                                      const T* __restrict__ Y_top, T* grad_top, int32_t cp) {
  for (int c = blockIdx.x * blockDim.x + threadIdx.x; c < cp; c += gridDim.x * blockDim.x) {
    float g0 = 0.f;
    for (int b = 0; b < batch; ++b) {
      const int r = head_rows[b];
      const float g = dh[(int64_t)b * dh_stride + c];
      if (r == 0) {
        g0 += g;
      } else {
        const bool on = Elem<T>::to_f32(Y_top[(int64_t)r * cp + c]) > 0.f;
        grad_top[(int64_t)r * cp + c] = on ? Elem<T>::from_f32(g) : Elem<T>::from_f32(0.f);
      }
    }
    grad_top[c] = (Elem<T>::to_f32(Y_top[c]) > 0.f) ? Elem<T>::from_f32(g0) : Elem<T>::from_f32(0.f);
  }
}

__global__ void __launch_bounds__(256) k_fill_zero(uint32_t* p, int64_t words) {
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < words; t += (int64_t)gridDim.x * blockDim.x)
    p[t] = 0u;
}

static int grid_for(int64_t items) { return (int)std::max<int64_t>(1, std::min<int64_t>((items + 255) / 256, 4096)); }

#define SSCN_DISPATCH(bf16, KERNEL, grid, block, ...)                                     \
  do {                                                                                    \
    if (bf16)                                                                             \
      hipLaunchKernelGGL(KERNEL<__bf16>, dim3(grid), dim3(block), 0, st, __VA_ARGS__);    \
    else                                                                                  \
      hipLaunchKernelGGL(KERNEL<float>, dim3(grid), dim3(block), 0, st, __VA_ARGS__);     \
  } while (0)

hipError_t launch_scatter_input(bool bf16, const void* feats, int32_t n, int32_t c_in, const int32_t* perm, void* X0,
                                int32_t cp0, hipStream_t st) {
  int grid = grid_for((int64_t)(n + 1) * cp0);
  if (bf16)
    hipLaunchKernelGGL(k_scatter_input<__bf16>, dim3(grid), dim3(256), 0, st, (const __bf16*)feats, n, c_in, perm,
                       (__bf16*)X0, cp0);
  else
    hipLaunchKernelGGL(k_scatter_input<float>, dim3(grid), dim3(256), 0, st, (const float*)feats, n, c_in, perm,
                       (float*)X0, cp0);
  return hipGetLastError();
}

hipError_t launch_gather_dfeats(bool bf16, const void* grad0, int32_t cp0, const int32_t* perm, int32_t n,
                                int32_t c_in, void* dfeats, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  int grid = grid_for((int64_t)n * c_in);
  if (bf16)
    hipLaunchKernelGGL(k_gather_dfeats<__bf16>, dim3(grid), dim3(256), 0, st, (const __bf16*)grad0, cp0, perm, n, c_in,
                       (__bf16*)dfeats);
  else
    hipLaunchKernelGGL(k_gather_dfeats<float>, dim3(grid), dim3(256), 0, st, (const float*)grad0, cp0, perm, n, c_in,
                       (float*)dfeats);
  return hipGetLastError();
}

hipError_t launch_pack(bool bf16, int mode, const void* W, int32_t A, int32_t c_in, int32_t c_out, int32_t cp_in,
                       int32_t cp_out, void* Bt, int32_t Npad, int32_t Kpad, hipStream_t st) {
  int grid = grid_for((int64_t)Npad * Kpad);
  if (bf16)
    hipLaunchKernelGGL(k_pack<__bf16>, dim3(grid), dim3(256), 0, st, mode, (const __bf16*)W, A, c_in, c_out, cp_in,
                       cp_out, (__bf16*)Bt, Npad, Kpad);
  else
    hipLaunchKernelGGL(k_pack<float>, dim3(grid), dim3(256), 0, st, mode, (const float*)W, A, c_in, c_out, cp_in,
                       cp_out, (float*)Bt, Npad, Kpad);
  return hipGetLastError();
}

hipError_t launch_softmax_xent(bool bf16, const float* logits, const int32_t* labels, int32_t batch, int32_t classes,
                               void* dlogits, int32_t dl_stride, float* loss_part, float* loss, hipStream_t st) {
  if (batch > 0) {
    if (bf16)
      hipLaunchKernelGGL(k_softmax_xent<__bf16>, dim3(batch), dim3(256), 0, st, logits, labels, batch, classes,
                         (__bf16*)dlogits, dl_stride, loss_part);
    else
      hipLaunchKernelGGL(k_softmax_xent<float>, dim3(batch), dim3(256), 0, st, logits, labels, batch, classes,
                         (float*)dlogits, dl_stride, loss_part);
  }
  hipLaunchKernelGGL(k_loss_final, dim3(1), dim3(64), 0, st, loss_part, batch, loss);
  return hipGetLastError();
}

hipError_t launch_head_scatter(bool bf16, const float* dh, int32_t dh_stride, const int32_t* head_rows,
                               int32_t batch, const void* Y_top, void* grad_top, int32_t cp, hipStream_t st) {
  int grid = (cp + 255) / 256;
  if (bf16)
    hipLaunchKernelGGL(k_head_scatter<__bf16>, dim3(grid), dim3(256), 0, st, dh, dh_stride, head_rows, batch,
                       (const __bf16*)Y_top, (__bf16*)grad_top, cp);
  else
    hipLaunchKernelGGL(k_head_scatter<float>, dim3(grid), dim3(256), 0, st, dh, dh_stride, head_rows, batch,
                       (const float*)Y_top, (float*)grad_top, cp);
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* p, int64_t bytes, hipStream_t st) {
  int64_t words = bytes / 4;
  if (words <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_zero, dim3(grid_for(words)), dim3(256), 0, st, (uint32_t*)p, words);
  return hipGetLastError();
}

}  // namespace sscn
