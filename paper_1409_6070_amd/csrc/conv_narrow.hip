// Forward of a sparse convolution with few input channels (Section 2.1: the
// first layer of a pen-stroke network has one input channel, of an image
// network three), on the vector ALUs.
//
// As a gather GEMM such a layer has K = A * Cp_in with Cp_in the channel count
// padded to a 16-byte vector, so a 3 x 3 window over one channel is 9 products
// per output in a K of 72 (128 after tile padding): the matrix cores would
// mostly multiply padding.  Here NARROW_SPLIT threads share an output row: each
// loads the row's window and its A input rows once, then computes every
// NARROW_SPLIT-th 16-byte output vector of the row with the weights staged in
// LDS as fp32 (read by broadcast), with the same bias-rectifier epilogue as the
// GEMM.
//
// With the pooling forward of the layer above (GemmArgs::pool_fwd) the rows
// are the pooling windows' slots 4 p + f, as in the GEMM's fused epilogue: four
// adjacent lanes take the four slots of one window (and the same share of its
// output vectors), each stores its convolution row (row 0 from window 0's slot
// 0 only), and per output vector the window's first maximum and its position
// are combined across the four lanes (earlier slots win ties) and stored by the
// slot-0 lane.

#include "common.h"
#include "epilogue.h"
#include "kernels.h"

#include <hip/hip_ext.h>

namespace sscn {

namespace {

typedef uint32_t nv4u __attribute__((ext_vector_type(4)));
constexpr int NARROW_AMAX = 9;   // largest window (3 x 3)
constexpr int NARROW_SPLIT = 2;  // threads per output row

template <int VE>
struct NarrowArg;
template <>
struct NarrowArg<8> {
  typedef uint64_t W;
};
template <>
struct NarrowArg<4> {
  typedef uint32_t W;
};

// The inputs of convolution row `row`: the first CIN channels of each of its
// window's input rows (zero for window positions f >= A), as fp32.  Every load
// is issued unconditionally (clamped index, selected value), so the window's
// loads go out together.
template <typename T, int CIN>
__device__ inline void narrow_inputs(const GemmArgs& a, int row, float (&xs)[NARROW_AMAX * CIN]) {
  const T* X = (const T*)a.src;
  const int* Rr = a.rmap + (int64_t)row * a.A;
  int q[NARROW_AMAX];
#pragma unroll
  for (int f = 0; f < NARROW_AMAX; ++f) {
    const int v = Rr[f < a.A ? f : a.A - 1];
    q[f] = f < a.A ? v : -1;
  }
#pragma unroll
  for (int f = 0; f < NARROW_AMAX; ++f) {
    const nv4u v = *(const nv4u*)(X + (int64_t)max(q[f], 0) * a.src_stride);
#pragma unroll
    for (int c = 0; c < CIN; ++c) xs[f * CIN + c] = q[f] >= 0 ? Elem<T>::to_f32(((const T*)&v)[c]) : 0.f;
  }
}

// Output vector n .. n + VE - 1 of a row with inputs xs: the products with the
// staged weights Wl[f * CIN + c][n] (zero rows for f >= A) summed in (f, c)
// order, then bias and rectifier.  Every lane of a wave reads the same weights
// (LDS broadcast).
template <typename T, int CIN>
__device__ inline nv4u narrow_vector(const GemmArgs& a, const float (&xs)[NARROW_AMAX * CIN], int n, const float* Wl,
                                     const float* bl, int ldw) {
  constexpr int VE = Elem<T>::VE;
  float s[VE];
#pragma unroll
  for (int e = 0; e < VE; ++e) s[e] = 0.f;
#pragma unroll
  for (int k = 0; k < NARROW_AMAX * CIN; ++k) {
    const float* w = Wl + k * ldw + n;
#pragma unroll
    for (int e = 0; e < VE; ++e) s[e] = fmaf(xs[k], w[e], s[e]);
  }
  nv4u o;
#pragma unroll
  for (int e = 0; e < VE; ++e) ((T*)&o)[e] = Elem<T>::from_f32(epi_value<T>(a, s[e], bl[n + e]));
  return o;
}

// One step of the first maximum over a window's slots: `late` (the later
// slots) replaces `early` element by element only where it is strictly greater,
// compared as fp32 exactly as the stored values convert; the argmax bytes follow
// the same choice.  Works on whole 32-bit words: a per-word select mask and one
// bit-select per word instead of per-element inserts.
template <typename T>
__device__ inline void first_max_step(const nv4u& early, const nv4u& late, typename NarrowArg<Elem<T>::VE>::W eam,
                                      typename NarrowArg<Elem<T>::VE>::W lam, nv4u& r,
                                      typename NarrowArg<Elem<T>::VE>::W& am) {
  typedef typename NarrowArg<Elem<T>::VE>::W AW;
  AW amask = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const uint32_t E = early[w], L = late[w];
    uint32_t m;
    if constexpr (Elem<T>::VE == 8) {  // two bf16 per word: element 2w low, 2w + 1 high
      const bool g0 = __uint_as_float(L << 16) > __uint_as_float(E << 16);
      const bool g1 = __uint_as_float(L & 0xffff0000u) > __uint_as_float(E & 0xffff0000u);
      m = (g0 ? 0x0000ffffu : 0u) | (g1 ? 0xffff0000u : 0u);
      amask |= (AW)((g0 ? 0x00ffu : 0u) | (g1 ? 0xff00u : 0u)) << (16 * w);
    } else {  // one fp32 per word
      const bool g = __uint_as_float(L) > __uint_as_float(E);
      m = g ? 0xffffffffu : 0u;
      amask |= (AW)(g ? 0xffu : 0u) << (8 * w);
    }
    r[w] = (L & m) | (E & ~m);
  }
  am = (lam & amask) | (eam & ~amask);
}

template <typename T, int CIN, bool POOL>
__global__ void __launch_bounds__(256) k_conv_narrow(GemmArgs a) {
  constexpr int VE = Elem<T>::VE;
  constexpr int KR = NARROW_AMAX * CIN;
  typedef typename NarrowArg<VE>::W AW;
  extern __shared__ float narrow_lds[];
  const int ldw = a.out_cols;
  float* Wl = narrow_lds;             // [KR][out_cols]
  float* bl = narrow_lds + KR * ldw;  // [out_cols]
  const T* Bt = (const T*)a.Bt;
  {
    // staged in groups of four per thread, the group's loads issued together
    const int total = (KR + 1) * ldw;
    for (int i0 = threadIdx.x; i0 < total; i0 += 4 * blockDim.x) {
      float v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = i0 + u * blockDim.x;
        const int k = i / ldw, n = i - k * ldw;
        const int f = k / CIN, c = k - f * CIN;
        const bool w_ok = i < total && k < KR && f < a.A && n < a.N;
        const bool b_ok = i < total && k == KR && n < a.N && a.bias;
        const T wv = Bt[w_ok ? (int64_t)n * a.Kpad + f * a.cseg + c : 0];
        const float bv = a.bias ? a.bias[b_ok ? n : 0] : 0.f;
        v[u] = w_ok ? Elem<T>::to_f32(wv) : b_ok ? bv : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (i0 + u * (int)blockDim.x < total) narrow_lds[i0 + u * blockDim.x] = v[u];
    }
  }
  __syncthreads();
  const int nvo = a.out_cols / VE;
  const int64_t rows = a.rows_dev ? (int64_t)(*a.rows_dev + a.rows_add) : (int64_t)a.rows_host;
  // NARROW_SPLIT threads per row, each taking every NARROW_SPLIT-th output
  // vector; POOL: rows counts the pooling windows, items are their slots
  // (slot fastest, so the four slots of a window sit in adjacent lanes)
  const int64_t items = rows * NARROW_SPLIT * (POOL ? 4 : 1);
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t it = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; it < items; it += stride) {
    float xs[KR];
    if constexpr (!POOL) {
      const int64_t m = it / NARROW_SPLIT;
      const int part = (int)(it - m * NARROW_SPLIT);
      narrow_inputs<T, CIN>(a, (int)m, xs);
      for (int v = part; v < nvo; v += NARROW_SPLIT) {
        const nv4u o = narrow_vector<T, CIN>(a, xs, v * VE, Wl, bl, ldw);
        *(nv4u*)((T*)a.out + m * a.out_stride + v * VE) = o;
      }
    } else {
      const int f = (int)(it & 3);
      const int64_t pp = it >> 2;
      const int64_t p = pp / NARROW_SPLIT;
      const int part = (int)(pp - p * NARROW_SPLIT);
      const int row = a.pslot[p * 4 + f];
      narrow_inputs<T, CIN>(a, row, xs);
      const bool store_row = row > 0 || (p == 0 && f == 0);
      for (int v = part; v < nvo; v += NARROW_SPLIT) {
        const int n = v * VE;
        nv4u o = narrow_vector<T, CIN>(a, xs, n, Wl, bl, ldw);
        if (store_row) *(nv4u*)((T*)a.out + (int64_t)row * a.out_stride + n) = o;
        // first maximum over the window's slots: adjacent pairs, then the
        // halves (a later slot wins only when strictly greater)
        AW am = 0;
#pragma unroll
        for (int e = 0; e < VE; ++e) am |= (AW)f << (8 * e);
#pragma unroll
        for (int d = 1; d <= 2; d <<= 1) {
          nv4u po;
#pragma unroll
          for (int w = 0; w < 4; ++w) po[w] = __shfl_xor(o[w], d, 64);
          AW pam;
          if constexpr (VE == 8) {
            const uint32_t lo = __shfl_xor((uint32_t)am, d, 64), hi = __shfl_xor((uint32_t)(am >> 32), d, 64);
            pam = ((AW)hi << 32) | lo;
          } else {
            pam = __shfl_xor(am, d, 64);
          }
          const bool upper = (f & d) != 0;  // this lane holds the later slots
          const nv4u early = upper ? po : o, late = upper ? o : po;
          const AW eam = upper ? pam : am, lam = upper ? am : pam;
          nv4u r;
          AW ram;
          first_max_step<T>(early, late, eam, lam, r, ram);
          o = r;
          am = ram;
        }
        if (f == 0) {
          *(nv4u*)((T*)a.pool_out + p * a.pool_stride + n) = o;
          *(AW*)(a.pool_argmax + p * a.pool_stride + n) = am;
        }
      }
    }
  }
}

// bf16: the same layer on the matrix cores.  A wave takes 16 GEMM rows at a
// time (pooling forward: four windows' slots, window-major) and every output
// channel in 16-wide blocks.  Its A operand is the rows' gathered inputs with
// k = f * CIN + c (A * CIN <= 32: one v_mfma_f32_16x16x32_bf16 step, zero
// past it), its B operand the weights of that k for each block's channels,
// loaded once per wave.  In the result lane (g, n) holds rows 4 g .. 4 g + 3 of
// channel n: with pooling, exactly one window's four slots, so the window's
// first maximum and its position are taken within the lane.  Non-pooled and
// pooled launches compute every row with the same operation, so their stored
// rows agree bit for bit.
constexpr int NARROW_NB = 8;  // at most 8 blocks of 16 output channels
#ifndef NARROW_MFMA_GRID
#define NARROW_MFMA_GRID 1280  // workgroups: about one round at five waves per SIMD
#endif

template <int CIN, bool POOL, int NBM>
__global__ void __launch_bounds__(256) k_conv_narrow_mfma(GemmArgs a) {
  typedef __bf16 T;
  typedef short s16x8 __attribute__((ext_vector_type(8)));
  const int lane = (int)threadIdx.x & 63;
  const int i = lane & 15, g = lane >> 4;
  const int A = a.A;
  const int nb = (a.out_cols + 15) / 16;
  const T* Bt = (const T*)a.Bt;
  const T* X = (const T*)a.src;
  // (32-bit offsets: the planner keeps every feature, window-list and weight
  // array of a layer below 2^31 elements)
  // The weights at k = f * CIN + c (zero past A * CIN) and the bias, staged in
  // LDS once per workgroup: rows of 32 k padded to 40 elements, so that the
  // 16 lanes reading one k group (16 channels, 16 bytes each) hit distinct banks.
  constexpr int LDW = 40;
  __shared__ __attribute__((aligned(16))) T wl[16 * NBM * LDW];
  __shared__ float bl[16 * NBM];
  // each wave's result rows, pooled rows and argmax bytes, staged for 16-byte stores
  constexpr int CW = 16 * NBM + 8;
  __shared__ __attribute__((aligned(16))) T cst[4][16 * CW];
  __shared__ __attribute__((aligned(16))) T pst[4][POOL ? 4 * CW : 8];
  __shared__ __attribute__((aligned(16))) uint8_t ast[4][POOL ? 4 * CW : 16];
  // weight and bias loads first; they reach LDS after the first rows' operand loads went out
  constexpr int WPT = 16 * NBM * 32 / 256;
  static_assert(WPT * 256 == 16 * NBM * 32, "whole weight tile per workgroup");
  T wv[WPT];
#pragma unroll
  for (int u = 0; u < WPT; ++u) {
    const int t = (int)threadIdx.x + 256 * u;
    const int n = t >> 5, k = t & 31, f = k / CIN, c = k - f * CIN;
    const bool ok = f < A && n < a.N;
    const T v = Bt[ok ? n * a.Kpad + f * a.cseg + c : 0];
    wv[u] = ok ? v : Elem<T>::from_f32(0.f);
  }
  const float bv = ((int)threadIdx.x < 16 * NBM && a.bias && (int)threadIdx.x < a.N) ? a.bias[threadIdx.x] : 0.f;
  const int64_t rows = a.rows_dev ? (int64_t)(*a.rows_dev + a.rows_add) : (int64_t)a.rows_host;
  const int64_t M = rows * (POOL ? 4 : 1);  // GEMM rows (pooling: the windows' slots)
  const int64_t waves = (int64_t)gridDim.x * (blockDim.x / 64);
  // this lane's A row of block blk (16 GEMM rows): its convolution row and its
  // inputs at k = 8 g .. 8 g + 7
  auto load_a = [&](int64_t blk, int& crow, bf16x8& av) {
    const int64_t m = blk * 16 + i;
    const bool live = m < M;
    crow = (int)m;
    if constexpr (POOL) crow = live ? a.pslot[m] : 0;
    if (!live) crow = 0;
    int idx[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int k = 8 * g + e, f = k / CIN;
      idx[e] = f < A ? a.rmap[crow * A + f] : 0;
    }
    s16x8 xa;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int k = 8 * g + e, f = k / CIN, c = k - f * CIN;
      const T v = X[idx[e] * a.src_stride + c];
      xa[e] = (f < A && live) ? __builtin_bit_cast(short, v) : (short)0;
    }
    av = __builtin_bit_cast(bf16x8, xa);
  };
  int64_t blk = (int64_t)blockIdx.x * (blockDim.x / 64) + ((int)threadIdx.x >> 6);
  int crow_n = 0;
  bf16x8 av_n{};
  if (blk * 16 < M) load_a(blk, crow_n, av_n);
#pragma unroll
  for (int u = 0; u < WPT; ++u) {
    const int t = (int)threadIdx.x + 256 * u;
    wl[(t >> 5) * LDW + (t & 31)] = wv[u];
  }
  if ((int)threadIdx.x < 16 * NBM) bl[threadIdx.x] = bv;
  __syncthreads();
  bf16x8 bw[NBM];
  float bias[NBM];
#pragma unroll
  for (int j = 0; j < NBM; ++j) {  // lane: channel 16 j + i, k = 8 g .. 8 g + 7
    bw[j] = *(const bf16x8*)(wl + (16 * j + i) * LDW + 8 * g);
    bias[j] = bl[16 * j + (lane & 15)];
  }
  for (; blk * 16 < M; blk += waves) {
    const int64_t m0 = blk * 16;
    const int crow = crow_n;
    const bf16x8 av = av_n;
    if ((blk + waves) * 16 < M) load_a(blk + waves, crow_n, av_n);  // the next block's loads during this one
    T* ct = cst[threadIdx.x >> 6];
#pragma unroll
    for (int j = 0; j < NBM; ++j) {
      if (j >= nb) break;
      const f32x4 d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bw[j], f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
      const int n = 16 * j + (lane & 15);
      T o[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) o[r] = Elem<T>::from_f32(epi_value<T>(a, d[r], bias[j]));
#pragma unroll
      for (int r = 0; r < 4; ++r) ct[(4 * g + r) * CW + n] = o[r];
      if constexpr (POOL) {  // first maximum over the window's slots (a later slot only when strictly greater)
        T mx = o[0];
        uint8_t am = 0;
#pragma unroll
        for (int r = 1; r < 4; ++r)
          if (Elem<T>::to_f32(o[r]) > Elem<T>::to_f32(mx)) {
            mx = o[r];
            am = (uint8_t)r;
          }
        pst[threadIdx.x >> 6][g * CW + n] = mx;
        ast[threadIdx.x >> 6][g * CW + n] = am;
      }
    }
    // (a wave's LDS operations run in order: the reads below see the writes above)
    const int nv = a.out_cols / 8;  // 16-byte vectors per row
#pragma unroll
    for (int it = 0; it < NBM / 2; ++it) {  // 16 rows x nv vectors, nv <= 2 NBM
      const int v = lane + 64 * it, row = min(v / nv, 15), cv = v - (v / nv) * nv;
      const int orr = __shfl(crow, row, 64);  // every lane takes part: the row's convolution row
      const int64_t mr = m0 + row;
      // pooling: every slot's convolution row, row 0 from window 0's slot 0 only
      if (v < 16 * nv && mr < M && (!POOL || orr > 0 || mr == 0))
        *(uint4*)((T*)a.out + orr * a.out_stride + 8 * cv) = *(const uint4*)(ct + row * CW + 8 * cv);
    }
    if constexpr (POOL) {
      const int w = lane / nv, cv = lane - w * nv;
      const int64_t p = (m0 >> 2) + w;
      if (lane < 4 * nv && 4 * p < M) {
        *(uint4*)((T*)a.pool_out + (int)p * a.pool_stride + 8 * cv) =
            *(const uint4*)(pst[threadIdx.x >> 6] + w * CW + 8 * cv);
        *(uint64_t*)(a.pool_argmax + (int)p * a.pool_stride + 8 * cv) =
            *(const uint64_t*)(ast[threadIdx.x >> 6] + w * CW + 8 * cv);
      }
    }
  }
}

typedef void (*NarrowKernel)(GemmArgs);
template <typename T, int CIN>
NarrowKernel narrow_kernel(bool pool) {
  return pool ? k_conv_narrow<T, CIN, true> : k_conv_narrow<T, CIN, false>;
}

}  // namespace

bool conv_narrow_ok(bool bf16, const GemmArgs& a, int cin) {
  const int VE = bf16 ? 8 : 4;
  return a.rmap && a.src && a.Bt && a.out && a.A >= 1 && a.A <= NARROW_AMAX && cin >= 1 && cin <= 4 && cin <= VE &&
         a.A * cin <= NARROW_KMAX && a.cseg >= VE && a.cseg % VE == 0 && a.src_stride % VE == 0 &&
         a.out_cols % VE == 0 && a.out_stride % VE == 0 && a.ksplit == 1 && !a.route && a.row_begin == 0 &&
         !a.x.kind && (a.epi == EPI_BIAS_RELU || a.epi == EPI_BIAS_LRELU) &&
         (size_t)(NARROW_AMAX * cin + 1) * a.out_cols * sizeof(float) <= 64 * 1024 &&
         (!a.pool_fwd || (a.pslot && a.pool_out && a.pool_argmax && a.rows_dev && a.pool_stride % VE == 0));
}

hipError_t launch_conv_narrow(bool bf16, const GemmArgs& in, int cin, int64_t max_rows, hipStream_t st) {
  if (!conv_narrow_ok(bf16, in, cin)) return hipErrorInvalidValue;
  GemmArgs a = in;
  // rows: pooling windows when pooling (max_rows counts their slots)
  if (a.pool_fwd) max_rows /= 4;
  if (max_rows <= 0) return hipSuccess;
  const int64_t items = max_rows * NARROW_SPLIT * (a.pool_fwd ? 4 : 1);
  // at most about eight workgroups per compute unit: each stages the weights once
  const int grid = (int)std::min<int64_t>(std::max<int64_t>((items + 255) / 256, 1), 2048);
  const size_t lds = (size_t)(NARROW_AMAX * cin + 1) * a.out_cols * sizeof(float);
  const bool pool = a.pool_fwd != 0;
  NarrowKernel kern = nullptr;
  switch (cin) {
    case 1: kern = bf16 ? narrow_kernel<__bf16, 1>(pool) : narrow_kernel<float, 1>(pool); break;
    case 2: kern = bf16 ? narrow_kernel<__bf16, 2>(pool) : narrow_kernel<float, 2>(pool); break;
    case 3: kern = bf16 ? narrow_kernel<__bf16, 3>(pool) : narrow_kernel<float, 3>(pool); break;
    default: kern = bf16 ? narrow_kernel<__bf16, 4>(pool) : narrow_kernel<float, 4>(pool); break;
  }
  if (bf16 && a.out_cols <= 16 * NARROW_NB && a.A * cin <= 32) {
    // matrix cores: one wave per 16 GEMM rows, at most eight waves per SIMD resident
    const int64_t rows16 = (max_rows * (pool ? 4 : 1) + 15) / 16;
    const int mgrid = (int)std::min<int64_t>(std::max<int64_t>((rows16 + 3) / 4, 1), NARROW_MFMA_GRID);
    NarrowKernel mk = nullptr;
    const bool w4 = a.out_cols <= 64;  // at most four channel blocks: fewer registers
#define SSCN_NARROW_PICK(C) \
  mk = pool ? (w4 ? k_conv_narrow_mfma<C, true, 4> : k_conv_narrow_mfma<C, true, NARROW_NB>) \
            : (w4 ? k_conv_narrow_mfma<C, false, 4> : k_conv_narrow_mfma<C, false, NARROW_NB>)
    switch (cin) {
      case 1: SSCN_NARROW_PICK(1); break;
      case 2: SSCN_NARROW_PICK(2); break;
      case 3: SSCN_NARROW_PICK(3); break;
      default: SSCN_NARROW_PICK(4); break;
    }
#undef SSCN_NARROW_PICK
    if (a.t_start || a.t_stop)
      hipExtLaunchKernelGGL(mk, dim3(mgrid), dim3(256), 0, st, a.t_start, a.t_stop, 0, a);
    else
      hipLaunchKernelGGL(mk, dim3(mgrid), dim3(256), 0, st, a);
    return hipGetLastError();
  }
  if (a.t_start || a.t_stop)
    hipExtLaunchKernelGGL(kern, dim3(grid), dim3(256), lds, st, a.t_start, a.t_stop, 0, a);
  else
    hipLaunchKernelGGL(kern, dim3(grid), dim3(256), lds, st, a);
  return hipGetLastError();
}

}  // namespace sscn
