// Input scatter, parameter packing, and the softmax output layer (Section 2.1:
// softmax on the output layer) with its cross-entropy loss.

#include "common.h"
#include "ground_tasks.h"
#include "kernels.h"

namespace sscn {

// X0[perm[i]][c] = feats[i][c] (zero padding columns); row 0 = 0, the input
// ground state.  One 16-byte vector of a row per item (cp0 is a multiple of
// the vector width); workgroup b of nb.
template <typename T>
__device__ inline void scatter_input_part(const T* __restrict__ feats, int32_t n, int32_t c_in,
                                          const int32_t* __restrict__ perm, T* X0, int32_t cp0, int b, int nb) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  constexpr int VE = Elem<T>::VE;
  const int nv = cp0 / VE;
  const int64_t total = (int64_t)(n + 1) * nv;
  for (int64_t t = (int64_t)b * blockDim.x + threadIdx.x; t < total; t += (int64_t)nb * blockDim.x) {
    const int64_t i = t / nv;
    const int c0 = (int)(t - i * nv) * VE;
    const int r = i == n ? 0 : perm[i];  // item n: the ground row
    if (i < n && r < 1) continue;        // rejected site
    u32x4 o;
#pragma unroll
    for (int e = 0; e < VE; ++e)
      ((T*)&o)[e] = (i < n && c0 + e < c_in) ? feats[i * c_in + c0 + e] : Elem<T>::from_f32(0.f);
    *(u32x4*)(X0 + (int64_t)r * cp0 + c0) = o;
  }
}

template <typename T>
__global__ void __launch_bounds__(256) k_scatter_input(const T* __restrict__ feats, int32_t n, int32_t c_in,
                                                       const int32_t* __restrict__ perm, T* X0, int32_t cp0) {
  scatter_input_part<T>(feats, n, c_in, perm, X0, cp0, blockIdx.x, gridDim.x);
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

// All weight packings of a step in one launch: one workgroup per tile of 64 n
// x 32 k of some job's output (tile_beg maps the flat block index to the job).
//   mode 0 (forward):   Bt[n][f*cp_in + c]  = W[(f*c_in + c)*c_out + n]
//     a transpose: the tile's 32 source rows are read along n (coalesced) into
//     LDS and written out along k;
//   mode 1 (backward):  Bt[c][f*cp_out + n] = W[(f*c_in + c)*c_out + n]
//     row segments: read and written along n.
// Entries outside the weight (padding) are zero.
constexpr int PACK_N = 64, PACK_K = 32;
template <typename T>
__global__ void __launch_bounds__(256) k_pack_all(PackArgs pa) {
  __shared__ T tile[PACK_K][PACK_N + 2];
  const T zero = Elem<T>::from_f32(0.f);
  const int own = (int)gridDim.x - pa.sc.blocks;
  if ((int)blockIdx.x >= own) {  // the input scatter's workgroups
    scatter_input_part<T>((const T*)pa.sc.feats, pa.sc.n, pa.sc.c_in, pa.sc.perm, (T*)pa.sc.X0, pa.sc.cp0,
                          (int)blockIdx.x - own, pa.sc.blocks);
    return;
  }
  for (int g = blockIdx.x; g < pa.tile_beg[pa.njobs]; g += own) {
    int ji = 0;
    while (ji + 1 < pa.njobs && g >= pa.tile_beg[ji + 1]) ++ji;
    const PackJob& j = pa.job[ji];
    const T* W = (const T*)j.W;
    T* Bt = (T*)j.Bt;
    const int tiles_k = j.Kpad / PACK_K;
    const int t = g - pa.tile_beg[ji];
    const int n0 = (t / tiles_k) * PACK_N, k0 = (t % tiles_k) * PACK_K;
    const float rcp_in = 1.f / (float)j.cp_in, rcp_out = 1.f / (float)j.cp_out;
    // every thread moves PACK_K * PACK_N / 256 elements; their loads are issued
    // together (clamped index, selected value), then stored
    constexpr int PER = PACK_K * PACK_N / 256;
    T v[PER];
    if (j.mode == 0) {
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int i = (int)threadIdx.x + u * 256;
        const int kk = i / PACK_N, nn = i % PACK_N;
        const int k = k0 + kk, n = n0 + nn;
        int f = (int)((float)k * rcp_in);  // k / cp_in: float estimate, exact correction
        f += (f + 1) * j.cp_in <= k ? 1 : 0;
        f -= f * j.cp_in > k ? 1 : 0;
        const int c = k - f * j.cp_in;
        const bool ok = f < j.A && c < j.c_in && n < j.c_out;
        const T w = W[ok ? ((int64_t)f * j.c_in + c) * j.c_out + n : 0];
        v[u] = ok ? w : zero;
      }
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int i = (int)threadIdx.x + u * 256;
        tile[i / PACK_N][i % PACK_N] = v[u];
      }
      __syncthreads();
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int i = (int)threadIdx.x + u * 256;
        const int nn = i / PACK_K, kk = i % PACK_K;
        Bt[(int64_t)(n0 + nn) * j.Kpad + k0 + kk] = tile[kk][nn];
      }
      __syncthreads();
    } else {
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int i = (int)threadIdx.x + u * 256;
        const int nn = i / PACK_K, kk = i % PACK_K;
        const int c = n0 + nn, k = k0 + kk;
        int f = (int)((float)k * rcp_out);
        f += (f + 1) * j.cp_out <= k ? 1 : 0;
        f -= f * j.cp_out > k ? 1 : 0;
        const int o = k - f * j.cp_out;
        const bool ok = f < j.A && o < j.c_out && c < j.c_in;
        const T w = W[ok ? ((int64_t)f * j.c_in + c) * j.c_out + o : 0];
        v[u] = ok ? w : zero;
      }
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int i = (int)threadIdx.x + u * 256;
        Bt[(int64_t)(n0 + i / PACK_K) * j.Kpad + k0 + i % PACK_K] = v[u];
      }
    }
  }
}

__device__ inline float wave_max(float v) {
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}
__device__ inline float wave_sum(float v) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// One workgroup per sample: softmax over the logits, the sample's loss term and
// dL/dlogits = (softmax - onehot) / batch.  Up to 4096 logits stay in registers.
template <typename T>
__global__ void __launch_bounds__(256) k_softmax_xent(const float* __restrict__ logits,
                                                      const int32_t* __restrict__ labels, int32_t batch,
                                                      int32_t classes, T* dlogits, int32_t dl_stride,
                                                      float* loss_part, float* loss, int32_t* counter,
                                                      int32_t* err) {
  constexpr int CACHE = 16;
  __shared__ float red[4];
  __shared__ int last;
  const int b = blockIdx.x, t = threadIdx.x, w = t >> 6;
  const float* z = logits + (int64_t)b * classes;
  float v[CACHE];
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < CACHE; ++i) {
    const int c = t + i * 256;
    v[i] = c < classes ? z[c] : -INFINITY;
    mx = fmaxf(mx, v[i]);
  }
  for (int c = t + CACHE * 256; c < classes; c += 256) mx = fmaxf(mx, z[c]);
  mx = wave_max(mx);
  if ((t & 63) == 0) red[w] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < CACHE; ++i) {
    v[i] = (t + i * 256 < classes) ? expf(v[i] - mx) : 0.f;
    s += v[i];
  }
  for (int c = t + CACHE * 256; c < classes; c += 256) s += expf(z[c] - mx);
  s = wave_sum(s);
  if ((t & 63) == 0) red[w] = s;
  __syncthreads();
  const float sum = (red[0] + red[1]) + (red[2] + red[3]);
  const int label = labels[b];
  const float inv_b = 1.f / (float)batch, inv_s = 1.f / sum;
  T* dl = dlogits + (int64_t)b * dl_stride;
#pragma unroll
  for (int i = 0; i < CACHE; ++i) {
    const int c = t + i * 256;
    if (c < dl_stride) dl[c] = Elem<T>::from_f32(c < classes ? (v[i] * inv_s - (c == label ? 1.f : 0.f)) * inv_b : 0.f);
  }
  for (int c = t + CACHE * 256; c < dl_stride; c += 256)
    dl[c] = Elem<T>::from_f32(c < classes ? (expf(z[c] - mx) * inv_s - (c == label ? 1.f : 0.f)) * inv_b : 0.f);
  // this sample's loss term; the last workgroup to finish sums all of them in
  // sample order (lane-strided, then a fixed butterfly) and resets the counter
  if (t == 0) {
    const bool ok = label >= 0 && label < classes;
    loss_part[b] = ok ? (logf(sum) + mx - z[label]) : 0.f;
    if (!ok) atomicOr(err, ERRBIT_LABEL);  // reported by the next sscn_layer_sizes
    __threadfence();
    last = atomicAdd(counter, 1) == batch - 1;
  }
  __syncthreads();
  if (!last || w != 0) return;
  __threadfence();
  float acc = 0.f;
  for (int i = t; i < batch; i += 64) acc += __hip_atomic_load(&loss_part[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  acc = wave_sum(acc);
  if (t == 0) {
    *loss = acc / (float)batch;
    __hip_atomic_store(counter, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

__global__ void k_loss_zero(float* loss) { *loss = 0.f; }

// Workgroup (x, p): 64 channels, samples 8p .. 8p+7; thread (channel c,
// sample lane l) takes samples 8p + l and 8p + l + 4; the four lanes are
// combined in LDS in a fixed order into partial p of each slot:
//   slot 0: sum of dh over empty samples (their top feature is the ground row),
//   slot 1: sum of the written delta rows (bias), slot 2+f: those whose window
//   position f reads the ground row.
// Row 0 of grad_top is set to zero (workgroups with p = 0): the final ground
// pass then finishes it as f'(Y_top[0]) * (0 + slot 0), the form it uses below
// a pooling layer.
template <typename T, int AC>
__global__ void __launch_bounds__(256) k_head_backward(HeadBwdArgs h, ExtraTask x) {
  if (run_extra<T>(x)) return;
  constexpr int J = 2 + AC;
  __shared__ float red[4][J][64];
  const int cl = threadIdx.x & 63, sl = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + cl;
  const int p = blockIdx.y;
  const T* Y = (const T*)h.Y_top;
  T* G = (T*)h.grad_top;
  float acc[J];
#pragma unroll
  for (int k = 0; k < J; ++k) acc[k] = 0.f;
  if (c < h.cp) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int b = p * 8 + sl + 4 * q;
      if (b >= h.batch) break;
      float g = 0.f;
      // unrolled so that several partials' loads are in flight; the sum keeps split order
#pragma unroll 4
      for (int ks = 0; ks < h.ksplit; ++ks) g += h.dh_part[ks * h.ks_stride + (int64_t)b * h.dh_stride + c];
      if (h.drop.on) g *= drop_factor(h.drop, (uint32_t)b, c);
      const int r = h.head_rows[b];
      if (r == 0) {
        acc[0] += g;
        continue;
      }
      const T v = Elem<T>::from_f32(g * act_factor(Elem<T>::to_f32(Y[(int64_t)r * h.cp + c]), h.slope));
      G[(int64_t)r * h.cp + c] = v;
      const float d = Elem<T>::to_f32(v);
      acc[1] += d;
#pragma unroll
      for (int f = 0; f < AC; ++f) acc[2 + f] += h.R[(int64_t)r * AC + f] == 0 ? d : 0.f;
    }
  }
#pragma unroll
  for (int k = 0; k < J; ++k) red[sl][k][cl] = acc[k];
  __syncthreads();
  if (sl != 0 || c >= h.cp) return;
  if (p == 0) G[c] = Elem<T>::from_f32(0.f);
#pragma unroll
  for (int k = 0; k < J; ++k)
    h.part[((int64_t)k * h.cp + c) * h.PM + p] = ((red[0][k][cl] + red[1][k][cl]) + red[2][k][cl]) + red[3][k][cl];
}

// Partials (sample chunks of 8) of the head backward.
int head_backward_parts(int32_t batch) { return std::max(1, (batch + 7) / 8); }

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
  int grid = grid_for((int64_t)(n + 1) * (cp0 / (bf16 ? 8 : 4)));
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

hipError_t launch_pack_all(bool bf16, const PackArgs& in, hipStream_t st) {
  PackArgs pa = in;
  int64_t total = 0;
  for (int i = 0; i < pa.njobs; ++i) {
    const PackJob& j = pa.job[i];
    // GEMM padding: N to a multiple of 64, K to a multiple of 32
    if (j.Npad % PACK_N || j.Kpad % PACK_K) return hipErrorInvalidValue;
    pa.tile_beg[i] = (int32_t)total;
    total += (int64_t)(j.Npad / PACK_N) * (j.Kpad / PACK_K);
  }
  if (pa.njobs <= 0 || total <= 0) return hipSuccess;
  if (total >= (1ll << 31)) return hipErrorInvalidValue;
  pa.tile_beg[pa.njobs] = (int32_t)total;
  if (pa.sc.X0) pa.sc.blocks = grid_for((int64_t)(pa.sc.n + 1) * (pa.sc.cp0 / (bf16 ? 8 : 4)));
  else pa.sc.blocks = 0;
  const int grid = (int)std::min<int64_t>(total, 16384) + pa.sc.blocks;  // one tile per workgroup up to 16384
  if (bf16)
    hipLaunchKernelGGL(k_pack_all<__bf16>, dim3(grid), dim3(256), 0, st, pa);
  else
    hipLaunchKernelGGL(k_pack_all<float>, dim3(grid), dim3(256), 0, st, pa);
  return hipGetLastError();
}

hipError_t launch_softmax_xent(bool bf16, const float* logits, const int32_t* labels, int32_t batch, int32_t classes,
                               void* dlogits, int32_t dl_stride, float* loss_part, float* loss, int32_t* counter,
                               int32_t* err, hipStream_t st) {
  if (batch > 0) {
    if (bf16)
      hipLaunchKernelGGL(k_softmax_xent<__bf16>, dim3(batch), dim3(256), 0, st, logits, labels, batch, classes,
                         (__bf16*)dlogits, dl_stride, loss_part, loss, counter, err);
    else
      hipLaunchKernelGGL(k_softmax_xent<float>, dim3(batch), dim3(256), 0, st, logits, labels, batch, classes,
                         (float*)dlogits, dl_stride, loss_part, loss, counter, err);
  } else {
    hipLaunchKernelGGL(k_loss_zero, dim3(1), dim3(1), 0, st, loss);
  }
  return hipGetLastError();
}

hipError_t launch_head_backward(bool bf16, const HeadBwdArgs& h, int32_t AC, hipStream_t st, const ExtraTask* extra) {
  const ExtraTask x = extra ? *extra : ExtraTask{};
  if (x.kind) return hipErrorInvalidValue;  // a 2-D grid: no extra workgroups
  const int P = head_backward_parts(h.batch);
  if (P > h.PM) return hipErrorInvalidValue;
  const dim3 grid((h.cp + 63) / 64, P);
#define SSCN_HEAD(T, A) hipLaunchKernelGGL((k_head_backward<T, A>), grid, dim3(256), 0, st, h, x)
  if (bf16) {
    switch (AC) {
      case 0: SSCN_HEAD(__bf16, 0); break;
      case 1: SSCN_HEAD(__bf16, 1); break;
      case 4: SSCN_HEAD(__bf16, 4); break;
      case 9: SSCN_HEAD(__bf16, 9); break;
      default: return hipErrorInvalidValue;
    }
  } else {
    switch (AC) {
      case 0: SSCN_HEAD(float, 0); break;
      case 1: SSCN_HEAD(float, 1); break;
      case 4: SSCN_HEAD(float, 4); break;
      case 9: SSCN_HEAD(float, 9); break;
      default: return hipErrorInvalidValue;
    }
  }
#undef SSCN_HEAD
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* p, int64_t bytes, hipStream_t st) {
  int64_t words = bytes / 4;
  if (words <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_zero, dim3(grid_for(words)), dim3(256), 0, st, (uint32_t*)p, words);
  return hipGetLastError();
}

}  // namespace sscn
