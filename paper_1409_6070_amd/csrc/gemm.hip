// The convolutions proper: dense contractions on CDNA4 matrix cores (MFMA).
//
// A sparse convolution (Section 2.3) computes, for every active output row o
// and for the ground row, b + sum_f W_f^T x_{R[o][f]}: a GEMM whose A operand
// is gathered row by row through the window lists.  The gather is fused into
// the LDS fill of the A tile (no gathered matrix is written to HBM); weights
// are packed once per step into [N][K] tiles and staged through LDS.
//
//  * forward      out = ReLU(G W + b)        rows: output sites + ground row
//  * input grad   dX  = sum_f delta[Rt[.][f]] W_f^T   rows: sites below
//  * softmax head logits = h W + b, dh = dlogits W^T  (window of one)
//  * weight grad  dW = G^T delta, split over sites; extra A rows produce
//                 db = sum delta and the ground-row sums D0[f] = sum over
//                 rows whose window position f reads the ground row.
//
// bf16: v_mfma_f32_16x16x32_bf16 (one per 32-wide k block);
// fp32: v_mfma_f32_16x16x4f32 (four per 16-wide k block).  Accumulation is
// always fp32.

#include "common.h"
#include "kernels.h"

namespace sscn {

template <typename T>
struct MfmaCore;

template <>
struct MfmaCore<__bf16> {
  static constexpr int KB = 32;  // k per block
  __device__ static inline void step(const __bf16* a_ptr, const __bf16* b_ptr, f32x4& acc) {
    bf16x8 a = *(const bf16x8*)a_ptr;
    bf16x8 b = *(const bf16x8*)b_ptr;
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
  }
};

template <>
struct MfmaCore<float> {
  static constexpr int KB = 16;
  __device__ static inline void step(const float* a_ptr, const float* b_ptr, f32x4& acc) {
    f32x4 a = *(const f32x4*)a_ptr;
    f32x4 b = *(const f32x4*)b_ptr;
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[0], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[1], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[2], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[3], acc, 0, 0, 0);
  }
};

// Tile shape: WM x WN waves, each TM x TN 16x16 MFMA tiles.
constexpr int G_WM = 2, G_WN = 2, G_TM = 2, G_TN = 2;
constexpr int G_THREADS = 64 * G_WM * G_WN;
constexpr int G_BM = G_WM * G_TM * 16;
constexpr int G_BN = G_WN * G_TN * 16;

template <typename T>
struct Tiles {
  static constexpr int VE = Elem<T>::VE;
  static constexpr int KB = MfmaCore<T>::KB;
  static constexpr int BK = 2 * KB;  // 128 bytes of k per LDS row
  static constexpr int LDK = BK + VE;  // padded LDS row (elements)
};

GemmTile gemm_tile(bool bf16) {
  return bf16 ? GemmTile{G_BM, G_BN, Tiles<__bf16>::BK} : GemmTile{G_BM, G_BN, Tiles<float>::BK};
}

// acc[i][j] += A_tile(wave rows i) * B_tile(wave cols j) over one BK slab in LDS
template <typename T>
__device__ inline void mma_slab(const T* As, const T* Bs, f32x4 (&acc)[G_TM][G_TN], int wm, int wn, int lane) {
  constexpr int LDK = Tiles<T>::LDK;
  constexpr int KB = Tiles<T>::KB;
  constexpr int VE = Tiles<T>::VE;
  const int r16 = lane & 15, g = lane >> 4;
#pragma unroll
  for (int kb = 0; kb < Tiles<T>::BK; kb += KB) {
#pragma unroll
    for (int i = 0; i < G_TM; ++i)
#pragma unroll
      for (int j = 0; j < G_TN; ++j)
        MfmaCore<T>::step(As + (wm * G_TM * 16 + i * 16 + r16) * LDK + kb + g * VE,
                          Bs + (wn * G_TN * 16 + j * 16 + r16) * LDK + kb + g * VE, acc[i][j]);
  }
}

template <typename T>
__global__ void __launch_bounds__(G_THREADS) k_gemm_gather(GemmArgs a) {
  constexpr int VE = Tiles<T>::VE;
  constexpr int BK = Tiles<T>::BK;
  constexpr int LDK = Tiles<T>::LDK;
  constexpr int KV = BK / VE;  // vectors per LDS row
  __shared__ __attribute__((aligned(16))) T As[G_BM * LDK];
  __shared__ __attribute__((aligned(16))) T Bs[G_BN * LDK];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / G_WN, wn = wave % G_WN;
  const int rows = a.rows_dev ? (*a.rows_dev + a.rows_add) : a.rows_host;
  const int span = rows - a.row_begin;
  if (span <= 0) return;
  const int tiles_m = (span + G_BM - 1) / G_BM;
  const int tiles_n = a.Npad / G_BN;
  const T* src = (const T*)a.src;
  const T* Bt = (const T*)a.Bt;

  for (int tile = blockIdx.x; tile < tiles_m * tiles_n; tile += gridDim.x) {
    const int tn = tile % tiles_n, tm = tile / tiles_n;
    const int m0 = a.row_begin + tm * G_BM, n0 = tn * G_BN;
    f32x4 acc[G_TM][G_TN];
#pragma unroll
    for (int i = 0; i < G_TM; ++i)
#pragma unroll
      for (int j = 0; j < G_TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int k0 = 0; k0 < a.Kpad; k0 += BK) {
      for (int v = tid; v < G_BM * KV; v += G_THREADS) {
        const int r = v / KV, kv = v - r * KV;
        const int m = m0 + r, k = k0 + kv * VE;
        Vec16 val = {{0u, 0u, 0u, 0u}};
        if (m < rows && k < a.K) {
          const int f = k / a.cseg, c = k - f * a.cseg;
          const int srow = a.rmap ? a.rmap[(int64_t)m * a.A + f] : m;
          if (srow >= 0) val = *(const Vec16*)(src + (int64_t)srow * a.src_stride + c);
        }
        *(Vec16*)(As + r * LDK + kv * VE) = val;
      }
      for (int v = tid; v < G_BN * KV; v += G_THREADS) {
        const int r = v / KV, kv = v - r * KV;
        *(Vec16*)(Bs + r * LDK + kv * VE) = *(const Vec16*)(Bt + (int64_t)(n0 + r) * a.Kpad + k0 + kv * VE);
      }
      __syncthreads();
      mma_slab<T>(As, Bs, acc, wm, wn, lane);
      __syncthreads();
    }

    const int g = lane >> 4, c16 = lane & 15;
#pragma unroll
    for (int i = 0; i < G_TM; ++i)
#pragma unroll
      for (int j = 0; j < G_TN; ++j) {
        const int n = n0 + wn * G_TN * 16 + j * 16 + c16;
        if (n >= a.out_cols) continue;
        const float bias = (a.bias && n < a.N) ? a.bias[n] : 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = m0 + wm * G_TM * 16 + i * 16 + g * 4 + r;
          if (m >= rows) continue;
          float v = acc[i][j][r] + bias;
          const int64_t o = (int64_t)m * a.out_stride + n;
          switch (a.epi) {
            case EPI_BIAS_RELU:
              ((T*)a.out)[o] = Elem<T>::from_f32(fmaxf(v, 0.f));
              break;
            case EPI_STORE:
              ((T*)a.out)[o] = Elem<T>::from_f32(v);
              break;
            default:
              ((float*)a.out)[o] = v;
              break;
          }
        }
      }
  }
}

template <typename T>
__global__ void __launch_bounds__(G_THREADS) k_wgrad(WGradArgs a) {
  constexpr int VE = Tiles<T>::VE;
  constexpr int BK = Tiles<T>::BK;
  constexpr int LDK = Tiles<T>::LDK;
  __shared__ __attribute__((aligned(16))) T As[G_BM * LDK];  // [m][site]
  __shared__ __attribute__((aligned(16))) T Bs[G_BN * LDK];  // [n][site]

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / G_WN, wn = wave % G_WN;
  const int rows = a.rows_dev ? (*a.rows_dev + a.rows_add) : a.rows_host;
  const int tiles_m = a.Mpad / G_BM, tiles_n = a.Npad / G_BN;
  const int ntiles = tiles_m * tiles_n * a.nchunks;
  const int per = ((rows + a.nchunks - 1) / a.nchunks + BK - 1) / BK * BK;
  const int m_gather = a.A * a.cseg;
  const T* src = (const T*)a.src;
  const T* dsrc = (const T*)a.dsrc;
  const T one = Elem<T>::from_f32(1.f), zero = Elem<T>::from_f32(0.f);

  for (int tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int tn = tile % tiles_n;
    const int tq = tile / tiles_n;
    const int tm = tq % tiles_m;
    const int chunk = tq / tiles_m;
    const int m0 = tm * G_BM, n0 = tn * G_BN;
    const int o_beg = chunk * per;
    const int o_end = min(rows, o_beg + per);
    f32x4 acc[G_TM][G_TN];
#pragma unroll
    for (int i = 0; i < G_TM; ++i)
#pragma unroll
      for (int j = 0; j < G_TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int ob = o_beg; ob < o_end; ob += BK) {
      // A^T slab: As[m][o - ob], gathered along m (contiguous channels of one row)
      for (int v = tid; v < BK * (G_BM / VE); v += G_THREADS) {
        const int ol = v / (G_BM / VE), mv = v - ol * (G_BM / VE);
        const int o = ob + ol, m = m0 + mv * VE;
        T vals[VE];
#pragma unroll
        for (int j = 0; j < VE; ++j) vals[j] = zero;
        if (o < o_end) {
          if (m < m_gather) {
            const int f = m / a.cseg, c = m - f * a.cseg;
            const int srow = a.rmap ? a.rmap[(int64_t)o * a.A + f] : o;
            Vec16 raw = *(const Vec16*)(src + (int64_t)srow * a.src_stride + c);
            const T* rv = (const T*)&raw;
#pragma unroll
            for (int j = 0; j < VE; ++j) vals[j] = rv[j];
          } else {
#pragma unroll
            for (int j = 0; j < VE; ++j) {
              const int mm = m + j;
              if (mm == a.m_ones) vals[j] = one;
              else if (a.m_ind >= 0 && mm >= a.m_ind && mm < a.m_ind + a.A)
                vals[j] = (a.rmap[(int64_t)o * a.A + (mm - a.m_ind)] == 0) ? one : zero;
            }
          }
        }
#pragma unroll
        for (int j = 0; j < VE; ++j) As[(mv * VE + j) * LDK + ol] = vals[j];
      }
      // B^T slab: Bs[n][o - ob]
      for (int v = tid; v < BK * (G_BN / VE); v += G_THREADS) {
        const int ol = v / (G_BN / VE), nv = v - ol * (G_BN / VE);
        const int o = ob + ol, n = n0 + nv * VE;
        T vals[VE];
#pragma unroll
        for (int j = 0; j < VE; ++j) vals[j] = zero;
        if (o < o_end && n < a.dsrc_cols) {
          Vec16 raw = *(const Vec16*)(dsrc + (int64_t)o * a.dsrc_stride + n);
          const T* rv = (const T*)&raw;
#pragma unroll
          for (int j = 0; j < VE; ++j) vals[j] = rv[j];
        }
#pragma unroll
        for (int j = 0; j < VE; ++j) Bs[(nv * VE + j) * LDK + ol] = vals[j];
      }
      __syncthreads();
      mma_slab<T>(As, Bs, acc, wm, wn, lane);
      __syncthreads();
    }

    float* part = a.part + (int64_t)chunk * a.Mpad * a.Npad;
    const int g = lane >> 4, c16 = lane & 15;
#pragma unroll
    for (int i = 0; i < G_TM; ++i)
#pragma unroll
      for (int j = 0; j < G_TN; ++j) {
        const int n = n0 + wn * G_TN * 16 + j * 16 + c16;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = m0 + wm * G_TM * 16 + i * 16 + g * 4 + r;
          part[(int64_t)m * a.Npad + n] = acc[i][j][r];
        }
      }
  }
}

__global__ void __launch_bounds__(256) k_wgrad_reduce(const float* __restrict__ part, int32_t nchunks, int32_t Mpad,
                                                      int32_t Npad, int32_t A, int32_t cseg, int32_t c_in,
                                                      int32_t c_out, int32_t m_ones, int32_t m_ind, float* dW,
                                                      float* db, float* D0) {
  const int m_gather = A * cseg;
  const int64_t total = (int64_t)Mpad * c_out;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += (int64_t)gridDim.x * blockDim.x) {
    const int m = (int)(t / c_out), n = (int)(t - (int64_t)m * c_out);
    float s = 0.f;
    for (int ch = 0; ch < nchunks; ++ch) s += part[((int64_t)ch * Mpad + m) * Npad + n];
    if (m < m_gather) {
      const int f = m / cseg, c = m - f * cseg;
      if (c < c_in) dW[((int64_t)f * c_in + c) * c_out + n] = s;
    } else if (m == m_ones) {
      if (db) db[n] = s;
    } else if (m_ind >= 0 && m >= m_ind && m < m_ind + A) {
      if (D0) D0[(int64_t)(m - m_ind) * c_out + n] = s;
    }
  }
}

template <typename T>
__global__ void __launch_bounds__(256) k_row0_dx(const T* __restrict__ W, const float* __restrict__ D0, int32_t A,
                                                 int32_t c_in, int32_t c_out, int32_t cp_in, T* grad_in) {
  __shared__ float red[256];
  const int c = blockIdx.x;
  float s = 0.f;
  if (c < c_in) {
    const int len = A * c_out;
    for (int t = threadIdx.x; t < len; t += blockDim.x) {
      const int f = t / c_out, n = t - f * c_out;
      s += Elem<T>::to_f32(W[((int64_t)f * c_in + c) * c_out + n]) * D0[t];
    }
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (threadIdx.x < off) red[threadIdx.x] += red[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0 && c < cp_in) grad_in[c] = Elem<T>::from_f32(red[0]);
}

static int device_grid_limit() { return 256 * 8; }

hipError_t launch_gemm(bool bf16, const GemmArgs& a, int64_t max_rows, hipStream_t st) {
  int64_t span = max_rows - a.row_begin;
  if (span <= 0) return hipSuccess;
  int64_t tiles = ((span + G_BM - 1) / G_BM) * (a.Npad / G_BN);
  int grid = (int)std::min<int64_t>(std::max<int64_t>(tiles, 1), device_grid_limit());
  if (bf16)
    hipLaunchKernelGGL(k_gemm_gather<__bf16>, dim3(grid), dim3(G_THREADS), 0, st, a);
  else
    hipLaunchKernelGGL(k_gemm_gather<float>, dim3(grid), dim3(G_THREADS), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_wgrad(bool bf16, const WGradArgs& a, hipStream_t st) {
  int64_t tiles = (int64_t)(a.Mpad / G_BM) * (a.Npad / G_BN) * a.nchunks;
  int grid = (int)std::min<int64_t>(std::max<int64_t>(tiles, 1), device_grid_limit());
  if (bf16)
    hipLaunchKernelGGL(k_wgrad<__bf16>, dim3(grid), dim3(G_THREADS), 0, st, a);
  else
    hipLaunchKernelGGL(k_wgrad<float>, dim3(grid), dim3(G_THREADS), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_wgrad_reduce(const float* part, int32_t nchunks, int32_t Mpad, int32_t Npad, int32_t A, int32_t cseg,
                               int32_t c_in, int32_t c_out, int32_t m_ones, int32_t m_ind, float* dW, float* db,
                               float* D0, hipStream_t st) {
  int64_t total = (int64_t)Mpad * c_out;
  int grid = (int)std::min<int64_t>((total + 255) / 256, 2048);
  hipLaunchKernelGGL(k_wgrad_reduce, dim3(std::max(grid, 1)), dim3(256), 0, st, part, nchunks, Mpad, Npad, A, cseg,
                     c_in, c_out, m_ones, m_ind, dW, db, D0);
  return hipGetLastError();
}

hipError_t launch_row0_dx(bool bf16, const void* W, const float* D0, int32_t A, int32_t c_in, int32_t c_out,
                          int32_t cp_in, void* grad_in, hipStream_t st) {
  if (bf16)
    hipLaunchKernelGGL(k_row0_dx<__bf16>, dim3(cp_in), dim3(256), 0, st, (const __bf16*)W, D0, A, c_in, c_out, cp_in,
                       (__bf16*)grad_in);
  else
    hipLaunchKernelGGL(k_row0_dx<float>, dim3(cp_in), dim3(256), 0, st, (const float*)W, D0, A, c_in, c_out, cp_in,
                       (float*)grad_in);
  return hipGetLastError();
}

}  // namespace sscn
