// Sparse 2x2 stride-2 max-pooling (Section 2.1) over active sites (Section 2.3).
//
// Forward: output row o takes, channel by channel, the maximum over the four
// rows its window reads (row 0, the ground row, for inactive locations) and
// records the first window position attaining it.  Row 0 passes the ground
// state through.
//
// Backward: windows do not overlap, so each active row below has exactly one
// window above and takes its gradient through that link (a gather, no
// atomics), with the ReLU mask of the convolution below applied in the same
// pass: the stored result is that convolution's output gradient delta.  Row 0
// (the ground row) sums the ground row above and every maximum an active
// window took from a ground location; it is reduced together with the
// convolution below's bias gradient and ground-row sums (block partials, then
// a fixed-order final pass: deterministic).

#include "common.h"
#include "ground_tasks.h"
#include "kernels.h"
#include "pool_route.h"

namespace sscn {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

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

// Sums over one block's rows for K slots at once: thread t holds acc[k][0..VE)
// for channel vector t % nv (the 256/nv row lanes of a vector are combined in
// a fixed order); the sum of slot k, channel e goes to out[k * slot_stride +
// e * PM].  Up to SB slots share one pass through LDS (red holds SB * 256 * VE
// floats): one barrier pair per pass, every (slot, channel) summed by one thread
// with independent LDS reads.
constexpr int SUM_SB = 6;
template <int VE, int K>
__device__ inline void block_channel_sums(const float (&acc)[K][VE], float* red, int nv, int cp, float* out,
                                          int64_t slot_stride, int PM) {
  const int t = threadIdx.x;
  const int lanes = 256 / nv;
#pragma unroll
  for (int k0 = 0; k0 < K; k0 += SUM_SB) {
#pragma unroll
    for (int kk = 0; kk < SUM_SB; ++kk)
      if (k0 + kk < K)
#pragma unroll
        for (int j = 0; j < VE; ++j) red[(kk * 256 + t) * VE + j] = acc[k0 + kk < K ? k0 + kk : 0][j];
    __syncthreads();
    const int kn = K - k0 < SUM_SB ? K - k0 : SUM_SB;
    for (int item = t; item < kn * cp; item += 256) {
      const int kk = item / cp, e = item - kk * cp;
      const int vv = e / VE, jj = e - vv * VE;
      const float* base = red + kk * 256 * VE + vv * VE + jj;
      float s = 0.f;
      for (int l = 0; l < lanes; ++l) s += base[l * nv * VE];
      out[(int64_t)(k0 + kk) * slot_stride + (int64_t)e * PM] = s;
    }
    __syncthreads();
  }
}

// Pooling backward fused with the sums of the convolution below (each row as
// in pool_route_item), one pass over the pooling layer's rows o >= 1: thread
// (lane l, channel vector v) of block b takes rows 1 + b*lanes + l, then every
// gridDim*lanes-th.  Partial p = block b of slot k, channel c:
// part[(k * cp + c) * PM + b].
template <typename T, int AC>
__global__ void __launch_bounds__(256) k_pool_bwd(GroundArgs g, ExtraTask x) {
  if (run_extra<T>(x)) return;
  constexpr int VE = Elem<T>::VE;
  constexpr int J = 2 + AC;
  __shared__ float red[SUM_SB * 256 * VE];
  const int nv = g.cp / VE;
  const int lanes = 256 / nv;
  const int t = threadIdx.x;
  const int v = t % nv, rl = t / nv;
  const int c = v * VE;
  const T* dY = (const T*)g.dY;
  const int n = *g.n_pool;
  float acc[J][VE];
#pragma unroll
  for (int k = 0; k < J; ++k)
#pragma unroll
    for (int j = 0; j < VE; ++j) acc[k][j] = 0.f;
  if (rl < lanes) {
#pragma unroll 1
    for (int o = 1 + blockIdx.x * lanes + rl; o <= n; o += own_grid(x) * lanes) {
      const u32x4 gv = *(const u32x4*)(dY + (int64_t)o * g.stride + c);
      pool_route_item<T, AC>(g, o, c, (const T*)&gv, acc);
    }
  }
  block_channel_sums<VE, J>(acc, red, nv, g.cp, g.part + blockIdx.x, (int64_t)g.cp * g.PM, g.PM);
}

// Partial sums behind a convolution's bias gradient and ground-row sums, and
// behind the ground row of a pooling layer above it.  Slots (per channel):
//   0       sum over pooling rows o >= 1 of dY[o] where the maximum came from a
//           ground location (blocks [0, B1), only with a pooling layer above);
//   1       sum over delta rows i >= 1 (bias gradient);
//   2 + f   sum over delta rows i >= 1 whose window position f reads the
//           ground row (D0[f]), f < AC.
// Row 0 of delta enters in the final pass.  A block takes a contiguous range of
// rows; partial p of slot k, channel c is part[(k * cp + c) * PM + p].
template <typename T, int AC>
__global__ void __launch_bounds__(256) k_ground_sums(GroundArgs g, ExtraTask x) {
  if (run_extra<T>(x)) return;
  constexpr int VE = Elem<T>::VE;
  typedef typename ArgPack<VE>::W AW;
  __shared__ float red[SUM_SB * 256 * VE];
  const int nv = g.cp / VE;
  const int lanes = 256 / nv;
  const int t = threadIdx.x;
  const int v = t % nv, rl = t / nv;
  const int c = v * VE;
  const bool active = rl < lanes;
  if ((int)blockIdx.x < g.B1) {
    const T* dY = (const T*)g.dY;
    const int n = *g.n_pool;
    const int per = (n + g.B1 - 1) / g.B1;
    const int o_beg = 1 + blockIdx.x * per, o_end = min(n + 1, o_beg + per);
    float acc[VE];
#pragma unroll
    for (int j = 0; j < VE; ++j) acc[j] = 0.f;
    if (active) {
#pragma unroll 4
      for (int o = o_beg + rl; o < o_end; o += lanes) {
        const i32x4 r = *(const i32x4*)(g.Rp + (int64_t)o * 4);
        const AW am = *(const AW*)(g.argmax + (int64_t)o * g.stride + c);
        const u32x4 gv = *(const u32x4*)(dY + (int64_t)o * g.stride + c);
#pragma unroll
        for (int j = 0; j < VE; ++j) {
          const int f = (int)((am >> (8 * j)) & 3);
          const int rf = f == 0 ? r.x : (f == 1 ? r.y : (f == 2 ? r.z : r.w));
          acc[j] += rf == 0 ? Elem<T>::to_f32(((const T*)&gv)[j]) : 0.f;
        }
      }
    }
    float acc1[1][VE];
#pragma unroll
    for (int j = 0; j < VE; ++j) acc1[0][j] = acc[j];
    block_channel_sums<VE, 1>(acc1, red, nv, g.cp, g.part + blockIdx.x, (int64_t)g.cp * g.PM, g.PM);
    return;
  }
  const int b = blockIdx.x - g.B1;
  const T* dZ = (const T*)g.dZ;
  const int n = *g.n_rows;
  const int per = (n + g.B2 - 1) / g.B2;
  const int i_beg = 1 + b * per, i_end = min(n + 1, i_beg + per);
  float acc[1 + AC][VE];
#pragma unroll
  for (int k = 0; k <= AC; ++k)
#pragma unroll
    for (int j = 0; j < VE; ++j) acc[k][j] = 0.f;
  if (active) {
#pragma unroll 4
    for (int i = i_beg + rl; i < i_end; i += lanes) {
      const u32x4 gv = *(const u32x4*)(dZ + (int64_t)i * g.stride + c);
      const WinRow<AC> wr = load_win_row<AC>(g.R, i);
#pragma unroll
      for (int j = 0; j < VE; ++j) {
        const float d = Elem<T>::to_f32(((const T*)&gv)[j]);
        acc[0][j] += d;
#pragma unroll
        for (int k = 0; k < AC; ++k) acc[1 + k][j] += wr.v[k] == 0 ? d : 0.f;
      }
    }
  }
  block_channel_sums<VE, 1 + AC>(acc, red, nv, g.cp, g.part + (int64_t)g.cp * g.PM + b, (int64_t)g.cp * g.PM, g.PM);
}

// Final pass: one workgroup per channel (ground_final_block).
template <typename T, int AC>
__global__ void __launch_bounds__(256) k_ground_final(GroundArgs g, ExtraTask x) {
  if (run_extra<T>(x)) return;
  ground_final_block<T, AC>(g, blockIdx.x);
}

// An extra task as its own launch.
template <typename T>
__global__ void __launch_bounds__(256) k_extra(ExtraTask x) { run_extra<T>(x); }

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

// kind 0: sums over delta rows (and pooling rows), then the final pass;
// kind 1: the fused pooling backward (B1 == B2 blocks);
// kind 2: the final pass alone (partials already written);
// kind 3: the sums alone.  The extra task rides on the first kernel of the call.
template <typename T, int AC>
static void launch_ground_t(const GroundArgs& g, int kind, hipStream_t st, const ExtraTask& x) {
  const ExtraTask none{};
  const int xb = x.kind ? x.blocks : 0;
  if (kind == 0 || kind == 3)
    hipLaunchKernelGGL((k_ground_sums<T, AC>), dim3(g.B1 + g.B2 + xb), dim3(256), 0, st, g, x);
  if (kind == 1) hipLaunchKernelGGL((k_pool_bwd<T, AC>), dim3(g.B2 + xb), dim3(256), 0, st, g, x);
  if (kind == 0 || kind == 2)
    hipLaunchKernelGGL((k_ground_final<T, AC>), dim3(g.cp + (kind == 2 ? xb : 0)), dim3(256), 0, st, g,
                       kind == 2 ? x : none);
}

static bool extra_ok(const ExtraTask& x) {
  if (x.kind == 0) return true;
  if (x.blocks < 1 || x.kind < 1 || x.kind > 3) return false;
  return x.kind == 2 || x.AC == 0 || x.AC == 1 || x.AC == 4 || x.AC == 9;
}

hipError_t launch_ground(bool bf16, const GroundArgs& g, int32_t AC, int kind, hipStream_t st,
                         const ExtraTask* extra) {
  if (g.B2 < 1 || g.B1 < 0 || g.B1 > g.PM || g.B2 > g.PM) return hipErrorInvalidValue;
  if (kind == 1 && (g.B1 != g.B2 || !g.X_pool || (AC == 4 && !g.gmask) || (AC != 0 && AC != 4 && !g.R)))
    return hipErrorInvalidValue;
  const ExtraTask x = extra ? *extra : ExtraTask{};
  if (!extra_ok(x)) return hipErrorInvalidValue;
#define SSCN_GROUND(T, A) launch_ground_t<T, A>(g, kind, st, x)
  if (bf16) {
    switch (AC) {
      case 0: SSCN_GROUND(__bf16, 0); break;
      case 1: SSCN_GROUND(__bf16, 1); break;
      case 4: SSCN_GROUND(__bf16, 4); break;
      case 9: SSCN_GROUND(__bf16, 9); break;
      default: return hipErrorInvalidValue;
    }
  } else {
    switch (AC) {
      case 0: SSCN_GROUND(float, 0); break;
      case 1: SSCN_GROUND(float, 1); break;
      case 4: SSCN_GROUND(float, 4); break;
      case 9: SSCN_GROUND(float, 9); break;
      default: return hipErrorInvalidValue;
    }
  }
#undef SSCN_GROUND
  return hipGetLastError();
}

hipError_t launch_extra(bool bf16, const ExtraTask& x, hipStream_t st) {
  if (x.kind == 0) return hipSuccess;
  if (!extra_ok(x)) return hipErrorInvalidValue;
  if (bf16)
    hipLaunchKernelGGL(k_extra<__bf16>, dim3(x.blocks), dim3(256), 0, st, x);
  else
    hipLaunchKernelGGL(k_extra<float>, dim3(x.blocks), dim3(256), 0, st, x);
  return hipGetLastError();
}

}  // namespace sscn
