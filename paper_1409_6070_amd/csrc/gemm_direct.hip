// Gather GEMM with MFMA operands loaded straight from memory (bf16).
//
// The operand layout of v_mfma_f32_16x16x32_bf16 is 8 consecutive k of one row
// per lane (lane l: row l % 16, k 8 * (l / 16) .. + 7) for both A and B.  With
// channels padded to multiples of 8 those 16 bytes are contiguous in the
// gathered input row (A = the window's rows, Section 2.3) and in the packed
// weights Bt[n][k], so each lane issues one 16-byte load per operand and k
// block -- no LDS staging and no barrier in the K loop.  A workgroup of SK
// waves computes one 32 x 64 output tile; wave w sums its own contiguous K
// range, four k blocks of loads in flight at a time, and the partial sums meet
// in LDS (in wave order, so the result is deterministic) for the epilogue,
// which writes 16-byte vectors.

#include "common.h"
#include "epilogue.h"
#include "ground_tasks.h"
#include "pool_route.h"
#include "kernels.h"

#include <hip/hip_ext.h>

#include <type_traits>

namespace sscn {

typedef uint32_t v4u __attribute__((ext_vector_type(4)));

constexpr int DIR_AMAX = 9;  // largest window (3x3)

// k / d for 0 <= k < 2^20, 1 <= d < 2^16: float estimate, then exact correction
__device__ inline int dir_div(int k, int d, float rcp) {
  int q = (int)((float)k * rcp);
  q += (q + 1) * d <= k ? 1 : 0;
  q -= q * d > k ? 1 : 0;
  return q;
}

// Epilogue in 16-byte vectors (8 columns of one row, the waves' partial sums
// added in wave order), thread t keeping column group c8e.  AC >= 0: the
// pooling backward of every row m >= 1 as well, and the tile's slot partial
// sums as partial tm (through red, reused).
struct NoPrefetch {};
template <int AC, bool PRE>
using PrefetchT = typename std::conditional<PRE, RouteIn<__bf16, AC < 0 ? 0 : AC>, NoPrefetch>::type;

template <int SK, int RP, int AC, bool PRE, int LDSF>
__device__ inline void store_vectors(const GemmArgs& a, float (*red)[DIRECT_BM][RP], const float (&bias8)[8], int c8e,
                                     int m0, int n0, int tm, int rows, const PrefetchT<AC, PRE>& pre) {
  typedef __bf16 T;
  constexpr int BM = DIRECT_BM, BN = DIRECT_BN, NT = 64 * SK, NV = BN / 8;
  constexpr int J = AC >= 0 ? 2 + AC : 1;
  static_assert(NT % NV == 0, "each thread keeps one column group");
  float acc[J][8];
  if constexpr (AC >= 0) {
#pragma unroll
    for (int k = 0; k < J; ++k)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[k][e] = 0.f;
  }
  for (int v = threadIdx.x; v < BM * NV; v += NT) {
    const int r = v / NV, c8 = c8e;
    const int m = m0 + r, n = n0 + c8;
    if (m >= rows || n >= a.out_cols) continue;
    float s[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) s[e] = 0.f;
#pragma unroll
    for (int q = 0; q < SK; ++q) {
      const f32x4 lo = *(const f32x4*)&red[q][r][c8], hi = *(const f32x4*)&red[q][r][c8 + 4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s[e] += lo[e];
        s[4 + e] += hi[e];
      }
    }
    v4u o;
    v4u y{0u, 0u, 0u, 0u};
    if (a.epi == EPI_STORE_MASK) y = *(const v4u*)((const T*)a.mask + (int64_t)m * a.mask_stride + n);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float v8 = epi_value<T>(a, s[e], bias8[e]);
      if (a.epi == EPI_STORE_MASK) v8 *= act_factor(Elem<T>::to_f32(((const T*)&y)[e]), a.slope);
      ((T*)&o)[e] = Elem<T>::from_f32(v8);
    }
    *(v4u*)((T*)a.out + (int64_t)m * a.out_stride + n) = o;
    if constexpr (AC >= 0) {
      if (m >= 1) {
        if constexpr (PRE)  // this thread's only row, its loads issued earlier
          route_apply<T, AC>(a.pr, n, pre, (const T*)&o, acc);
        else
          pool_route_item<T, AC>(a.pr, m, n, (const T*)&o, acc);
      }
    }
  }
  if constexpr (AC >= 0) tile_slot_sums<8, J, NT, NV, LDSF>(acc, &red[0][0][0], a.pr, n0, tm);
}

// Pooling forward in the epilogue (GemmArgs::pool_fwd): the tile's rows are
// the slots 4 p + f of pooling windows p.  Each thread forms its 16-byte
// vectors as the plain epilogue does, stores the slot's convolution row (row 0
// from slot 0 only) and stages the vector in LDS; then the first maximum over
// each window's four slots, per channel, goes to the pooling layer with its
// position.
template <int SK, int RP>
__device__ inline void store_pooled_direct(const GemmArgs& a, float (*red)[DIRECT_BM][RP], const float (&bias8)[8],
                                           int c8e, int m0, int n0, int rows, const int32_t* Cr) {
  typedef __bf16 T;
  constexpr int BM = DIRECT_BM, BN = DIRECT_BN, NT = 64 * SK, NV = BN / 8, SP = BN + 8;
  typedef typename ArgPack<8>::W AW;
  __shared__ __attribute__((aligned(16))) T Ps[BM * SP];  // the tile's stored values
  for (int v = threadIdx.x; v < BM * NV; v += NT) {
    const int r = v / NV, c8 = c8e;
    const int m = m0 + r, n = n0 + c8;
    if (m >= rows || n >= a.out_cols) continue;
    float s[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) s[e] = 0.f;
#pragma unroll
    for (int q = 0; q < SK; ++q) {
      const f32x4 lo = *(const f32x4*)&red[q][r][c8], hi = *(const f32x4*)&red[q][r][c8 + 4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s[e] += lo[e];
        s[4 + e] += hi[e];
      }
    }
    v4u o;
#pragma unroll
    for (int e = 0; e < 8; ++e) ((T*)&o)[e] = Elem<T>::from_f32(epi_value<T>(a, s[e], bias8[e]));
    const int row = Cr[r];
    if (row > 0 || m == 0) *(v4u*)((T*)a.out + (int64_t)row * a.out_stride + n) = o;
    *(v4u*)(Ps + r * SP + c8) = o;
  }
  __syncthreads();
  for (int v = threadIdx.x; v < (BM / 4) * NV; v += NT) {
    const int pr = v / NV, c8 = (v - pr * NV) * 8;
    const int m = m0 + 4 * pr, n = n0 + c8;
    if (m >= rows || n >= a.out_cols) continue;
    // running first maximum over the four slots (one staged vector at a time)
    v4u out = *(const v4u*)(Ps + (4 * pr) * SP + c8);
    AW am = 0;
#pragma unroll
    for (int f = 1; f < 4; ++f) {
      const v4u in = *(const v4u*)(Ps + (4 * pr + f) * SP + c8);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const bool gt = Elem<T>::to_f32(((const T*)&in)[j]) > Elem<T>::to_f32(((const T*)&out)[j]);
        if (gt) {
          ((T*)&out)[j] = ((const T*)&in)[j];
          am = (am & ~((AW)0xff << (8 * j))) | ((AW)f << (8 * j));
        }
      }
    }
    const int64_t p = m / 4;
    *(v4u*)((T*)a.pool_out + p * a.pool_stride + n) = out;
    *(AW*)(a.pool_argmax + p * a.pool_stride + n) = am;
  }
}

template <int SK, int RAC>
__global__ void __launch_bounds__(64 * SK) k_gemm_direct(GemmArgs a) {
  typedef __bf16 T;
  constexpr int TM = DIRECT_BM / 16, TN = DIRECT_BN / 16;
  constexpr int BM = DIRECT_BM, BN = DIRECT_BN, NT = 64 * SK;
  constexpr int CH = 3;        // k blocks (32 k each) of loads in flight per wave
  constexpr int RP = BN + 4;   // LDS pitch of the partial sums (floats)
  constexpr bool POOL = RAC == POOL_FWD_MODE;
  __shared__ int32_t Rs[BM * DIR_AMAX];
  // the waves' partial sums; with the pooling backward also every slot sum of
  // the tile at once (one pass through LDS)
  constexpr int REDF = SK * BM * RP, SLOTF = RAC >= 0 ? (2 + RAC) * NT * 8 : 0;
  constexpr int LDSF = REDF > SLOTF ? REDF : SLOTF;
  __shared__ __attribute__((aligned(16))) float red_lds[LDSF];
  float(*red)[BM][RP] = (float(*)[BM][RP])red_lds;
  __shared__ int32_t Cr[POOL ? BM : 1];  // pooling forward: the convolution row of each slot

  if (run_extra<T>(a.x)) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int rows_in = a.rows_dev ? *a.rows_dev : a.rows_host;
  const int tiles_n = a.Npad / BN;
  const int A = a.A;
  const int c8e = (tid % (BN / 8)) * 8;  // the column group this thread stores in the epilogue
  constexpr int RA = RAC < 0 ? 0 : RAC;
  // pooling backward in the epilogue with one row per thread (four waves):
  // that row's window, argmax, pooled values and ground mask before the K loop
  constexpr bool PRE = RAC >= 0 && NT == BM * (BN / 8);
  constexpr int EPT = (BM * DIR_AMAX + NT - 1) / NT;  // window entries per thread
  // A tile's window entries (the pooling forward: its slots' convolution rows)
  // for output rows m < bound.
  auto first_level = [&](int e, int m0, int bound) -> int {
    const int r = e / A, f = e - r * A, m = m0 + r;
    if (e >= BM * A || m >= bound) return -1;
    if constexpr (POOL) return a.pslot[m];
    return a.rmap ? a.rmap[(int64_t)m * A + f] : (f == 0 ? m : -1);
  };
  // The first tile's loads that do not need the row count are issued before it
  // arrives, bounded by the rows the grid was sized for (which every list and
  // row buffer holds): its window entries, its bias and its routing inputs.
  int first[EPT];
  float bias8[8];
  PrefetchT<RAC, PRE> pre;
  {
    const int m0 = a.row_begin + ((int)blockIdx.x / tiles_n) * BM, n0 = ((int)blockIdx.x % tiles_n) * BN;
#pragma unroll
    for (int i = 0; i < EPT; ++i) first[i] = first_level(tid + i * NT, m0, a.rows_cap);
    // (the pooling backward's launches are input gradients: no bias)
#pragma unroll
    for (int e = 0; e < 8; ++e)
      bias8[e] = (RAC < 0 && a.bias && n0 + c8e + e < a.N) ? a.bias[n0 + c8e + e] : 0.f;
    const int pre_m = m0 + tid / (BN / 8);
    if constexpr (PRE)
      if (pre_m >= 1 && pre_m < a.rows_cap && n0 + c8e < a.out_cols)
        route_load_window<T, RA>(a.pr, pre_m, n0 + c8e, pre);
  }
  const int rows = (rows_in + (a.rows_dev ? a.rows_add : 0)) * (POOL ? 4 : 1);
  const int span = rows - a.row_begin;
  if (span <= 0) return;
  const int tiles_m = (span + BM - 1) / BM;
  const int ntiles = tiles_m * tiles_n;
  const int ksteps = (a.K + 31) / 32;
  const int per = (ksteps + SK - 1) / SK;
  const int kb = min(ksteps, w * per), ke = min(ksteps, kb + per);
  const float rcp = 1.f / (float)a.cseg;
  const T* src = (const T*)a.src;
  const T* Bt = (const T*)a.Bt;

  const int grid = own_grid(a.x);
  for (int tile = blockIdx.x; tile < ntiles; tile += grid) {
    const int tn = tile % tiles_n, tm = tile / tiles_n;
    const int m0 = a.row_begin + tm * BM, n0 = tn * BN;
    const bool later = tile != (int)blockIdx.x;  // the first tile's loads were issued above
    if (later) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        bias8[e] = (RAC < 0 && a.bias && n0 + c8e + e < a.N) ? a.bias[n0 + c8e + e] : 0.f;
    }
    const int pre_m = m0 + tid / (BN / 8);
    const bool pre_on = PRE && pre_m >= 1 && pre_m < rows && n0 + c8e < a.out_cols;
    if constexpr (PRE)
      if (later && pre_on) route_load_window<T, RA>(a.pr, pre_m, n0 + c8e, pre);
#pragma unroll
    for (int i = 0; i < EPT; ++i) {  // the tile's window rows (-1: none)
      const int e = tid + i * NT;
      if (e < BM * A) {
        const int r = e / A, f = e - r * A;
        int v = -1;
        if (m0 + r < rows) {
          const int l1 = later ? first_level(e, m0, rows) : first[i];
          if constexpr (POOL) {  // l1 is the slot's convolution row
            if (f == 0) Cr[r] = l1;
            v = a.rmap ? a.rmap[(int64_t)l1 * A + f] : (f == 0 ? l1 : -1);
          } else {
            v = l1;
          }
        }
        Rs[e] = v;
      }
    }
    __syncthreads();

    f32x4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int k0 = kb; k0 < ke; k0 += CH) {
      v4u ra[CH][TM], rb[CH][TN];
#pragma unroll
      for (int c = 0; c < CH; ++c) {
        const int ks = k0 + c;
        if (ks < ke) {  // uniform over the wave
          const int k = ks * 32 + g * 8;
          const bool in_k = k < a.K;
          const int f = in_k ? dir_div(k, a.cseg, rcp) : 0;
          const int col = in_k ? k - f * a.cseg : 0;
#pragma unroll
          for (int i = 0; i < TM; ++i) {
            const int srow = in_k ? Rs[(i * 16 + r16) * A + f] : -1;
            const v4u val = *(const v4u*)(src + (int64_t)max(srow, 0) * a.src_stride + col);
            ra[c][i] = srow >= 0 ? val : v4u{0u, 0u, 0u, 0u};
          }
#pragma unroll
          for (int j = 0; j < TN; ++j)
            rb[c][j] = *(const v4u*)(Bt + (int64_t)(n0 + j * 16 + r16) * a.Kpad + ks * 32 + g * 8);
        }
      }
#pragma unroll
      for (int c = 0; c < CH; ++c) {
        if (k0 + c < ke) {
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ra[c][i]),
                                                                  __builtin_bit_cast(bf16x8, rb[c][j]), acc[i][j], 0,
                                                                  0, 0);
        }
      }
    }

    if constexpr (PRE)
      if (pre_on) route_load_children<T, RA>(a.pr, n0 + c8e, pre);
    // partial sums of every wave to LDS (MFMA output: lane holds rows 4g..4g+3 of column r16)
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[w][i * 16 + g * 4 + r][j * 16 + r16] = acc[i][j][r];
    __syncthreads();

    if constexpr (POOL) {
      store_pooled_direct<SK, RP>(a, red, bias8, c8e, m0, n0, rows, Cr);
    } else if (epi_stores_T(a.epi)) {
      store_vectors<SK, RP, RAC, PRE, LDSF>(a, red, bias8, c8e, m0, n0, tm, rows, pre);
    } else {
      for (int e = tid; e < BM * BN; e += NT) {
        const int r = e / BN, c = e - r * BN;
        const int m = m0 + r, n = n0 + c;
        if (m >= rows || n >= a.out_cols) continue;
        float s = 0.f;
#pragma unroll
        for (int q = 0; q < SK; ++q) s += red[q][r][c];
        store_out<T>(a, m, n, epi_value<T>(a, s, (a.bias && n < a.N) ? a.bias[n] : 0.f));
      }
    }
    __syncthreads();
  }
}

template <int SK>
static void launch_direct_sk(const GemmArgs& a, int64_t max_rows, hipStream_t st) {
  const int64_t span = max_rows - a.row_begin;
  const int64_t tiles = ((span + DIRECT_BM - 1) / DIRECT_BM) * (a.Npad / DIRECT_BN);
  const int grid = (int)std::min<int64_t>(std::max<int64_t>(tiles, 1), 2048) + (a.x.kind ? a.x.blocks : 0);
  void (*kern)(GemmArgs) = a.pool_fwd ? k_gemm_direct<SK, POOL_FWD_MODE>
                           : !a.route ? k_gemm_direct<SK, -1>
                           : a.route_ac == 4 ? k_gemm_direct<SK, 4>
                                             : k_gemm_direct<SK, 0>;
  if (a.t_start || a.t_stop)
    hipExtLaunchKernelGGL(kern, dim3(grid), dim3(64 * SK), 0, st, a.t_start, a.t_stop, 0, a);
  else
    hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * SK), 0, st, a);
}

hipError_t launch_gemm_direct(const GemmArgs& a, int64_t max_rows, hipStream_t st) {
  if (max_rows - a.row_begin <= 0) return hipSuccess;
  if (a.rows_cap != max_rows) return hipErrorInvalidValue;
  if (a.A < 1 || a.A > DIR_AMAX || a.cseg % 8 || a.src_stride % 8 || a.Npad % DIRECT_BN || a.Kpad % 32 ||
      a.Kpad < (a.K + 31) / 32 * 32 || a.ksplit != 1)
    return hipErrorInvalidValue;
  switch (a.sk) {
    case 1: launch_direct_sk<1>(a, max_rows, st); break;
    case 2: launch_direct_sk<2>(a, max_rows, st); break;
    case 4: launch_direct_sk<4>(a, max_rows, st); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace sscn
