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
  if (a.t_start || a.t_stop)
    hipExtLaunchKernelGGL(kern, dim3(grid), dim3(256), lds, st, a.t_start, a.t_stop, 0, a);
  else
    hipLaunchKernelGGL(kern, dim3(grid), dim3(256), lds, st, a);
  return hipGetLastError();
}

}  // namespace sscn
