// Backward of the sparse 2x2 stride-2 max-pooling (Section 2.1) for one
// pooling row and one 16-byte channel vector, shared by the pooling backward
// kernel and the gather-GEMM epilogue that produces the pooling layer's
// gradient, plus the fixed-order reduction of the per-thread slot sums of one
// GEMM output tile.
//
// Windows do not overlap, so each active row below has exactly one window above
// and takes its gradient through that link; the rectifier derivative of the
// convolution below is applied in the same step, so what is stored is that
// convolution's delta.  Slot sums (per channel) behind the convolution's bias
// gradient and ground-row chain:
//   0       pooling-row gradients whose maximum came from the ground row;
//   1       delta rows >= 1;
//   2 + f   delta rows >= 1 whose window position f reads the ground row.
#pragma once

#include "common.h"
#include "kernels.h"

namespace sscn {

typedef int32_t ri32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t ru32x4 __attribute__((ext_vector_type(4)));

// VE argmax bytes (VE = 8 or 4) as one integer load/store.
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

// Row i of a convolution's window list (AC entries; a 2x2 window as one vector).
template <int AC>
struct WinRow {
  int32_t v[AC > 0 ? AC : 1];
};
template <>
struct WinRow<4> {
  ri32x4 v;
};
template <int AC>
__device__ inline WinRow<AC> load_win_row(const int32_t* __restrict__ R, int64_t i) {
  WinRow<AC> w;
  if constexpr (AC == 4) {
    w.v = *(const ri32x4*)(R + i * 4);
  } else {
#pragma unroll
    for (int k = 0; k < AC; ++k) w.v[k] = R[i * AC + k];
  }
  return w;
}

// Pooling row o >= 1, channels c .. c+VE-1, with its stored gradient gv: the
// window's first maximum came from child row i = Rp[o][a] (a = argmax[o]),
// whose stored value it copies, so the rectifier derivative of the convolution
// below is read off the pooling output X_pool[o]:
//   i >= 1:  delta[i] = gv * f'(X_pool[o]), delta of the other children 0
//            (written: each child row lies in exactly one window), added to
//            slot 1 and, where the convolution's window position k of row i
//            reads the ground row (R[i][k] == 0), to slot 2 + k;
//   i == 0:  gv is added to slot 0.
// The ground pattern of the children's windows comes from the rulebook's
// child ground mask for AC == 4 and from the children's window rows for other
// AC.  The loads come in two steps that a caller may issue early: the row's
// window, argmax, pooled values (and mask), then (AC not 0 or 4 only) every
// child's window row.
template <int AC>
struct ChildWins {
  WinRow<AC> wr[4];
};
template <>
struct ChildWins<0> {};
template <>
struct ChildWins<4> {
  uint32_t gm;
};

template <typename T, int AC>
struct RouteIn {
  ri32x4 r;
  typename ArgPack<Elem<T>::VE>::W am;
  ru32x4 xp;
  ChildWins<AC> cw;
};

template <typename T, int AC>
__device__ inline void route_load_window(const GroundArgs& g, int64_t o, int c, RouteIn<T, AC>& q) {
  typedef typename ArgPack<Elem<T>::VE>::W AW;
  q.r = *(const ri32x4*)(g.Rp + o * 4);
  q.am = *(const AW*)(g.argmax + o * g.stride + c);
  q.xp = *(const ru32x4*)((const T*)g.X_pool + o * g.stride + c);
  if constexpr (AC == 4) q.cw.gm = g.gmask[o];
}

template <typename T, int AC>
__device__ inline void route_load_children(const GroundArgs& g, int c, RouteIn<T, AC>& q) {
  if constexpr (AC != 0 && AC != 4) {
#pragma unroll
    for (int f = 0; f < 4; ++f) q.cw.wr[f] = load_win_row<AC>(g.R, q.r[f]);
  }
}

template <typename T, int AC>
__device__ inline void route_apply(const GroundArgs& g, int c, const RouteIn<T, AC>& q, const T* gv,
                                   float (&acc)[2 + AC][Elem<T>::VE]) {
  constexpr int VE = Elem<T>::VE;
  T* dZ = (T*)g.dZ;
  // bit f: child f is the ground row; bit AC f + k: child f's window position k reads it
  const uint32_t gch = (q.r[0] == 0 ? 1u : 0u) | (q.r[1] == 0 ? 2u : 0u) | (q.r[2] == 0 ? 4u : 0u) |
                       (q.r[3] == 0 ? 8u : 0u);
  uint64_t gw = 0;
  if constexpr (AC == 4) {
    gw = q.cw.gm;
  } else if constexpr (AC > 0) {
#pragma unroll
    for (int f = 0; f < 4; ++f)
#pragma unroll
      for (int k = 0; k < AC; ++k) gw |= (uint64_t)(q.cw.wr[f].v[k] == 0 ? 1u : 0u) << (AC * f + k);
  }
  ru32x4 out[4];
  // every sum is updated on both branches (a select, not a branch), so that
  // the accumulators stay in registers
#pragma unroll
  for (int j = 0; j < VE; ++j) {
    const int a = (int)((q.am >> (8 * j)) & 3);
    const float gj = Elem<T>::to_f32(gv[j]);
    const T o = Elem<T>::from_f32(gj * act_factor(Elem<T>::to_f32(((const T*)&q.xp)[j]), g.slope));
    const bool ground = (gch >> a) & 1u;
    const float d = ground ? 0.f : Elem<T>::to_f32(o);
    acc[0][j] += ground ? gj : 0.f;
    acc[1][j] += d;
    if constexpr (AC > 0) {
      const uint64_t ga = gw >> (AC * a);
#pragma unroll
      for (int k = 0; k < AC; ++k) acc[2 + k][j] += ((ga >> k) & 1u) ? d : 0.f;
    }
#pragma unroll
    for (int f = 0; f < 4; ++f) ((T*)&out[f])[j] = a == f ? o : Elem<T>::from_f32(0.f);
  }
#pragma unroll
  for (int f = 0; f < 4; ++f)
    if (q.r[f] != 0) *(ru32x4*)(dZ + (int64_t)q.r[f] * g.stride + c) = out[f];
}

template <typename T, int AC>
__device__ inline void pool_route_item(const GroundArgs& g, int64_t o, int c, const T* gv,
                                       float (&acc)[2 + AC][Elem<T>::VE]) {
  RouteIn<T, AC> q;
  route_load_window<T, AC>(g, o, c, q);
  route_load_children<T, AC>(g, c, q);
  route_apply<T, AC>(g, c, q, gv, acc);
}

// Slot sums of one GEMM output tile: thread t holds acc for channel vector
// t % NV of the tile (NV vectors of VE channels from n0) over its rows.  Up to
// LDSF / (NT * VE) slots at a time go through lds (LDSF floats); each
// (slot, channel) is then summed by one thread over the NT / NV threads of its
// vector in thread order, and part[(k * cp + c) * PM + tm] receives slot k of
// channel c < cp.  All threads of the block call it; it synchronises before
// its first use of lds, and the caller before reusing lds.
template <int VE, int J, int NT, int NV, int LDSF>
__device__ inline void tile_slot_sums(const float (&acc)[J][VE], float* lds, const GroundArgs& g, int n0, int tm) {
  typedef float f4 __attribute__((ext_vector_type(4)));
  constexpr int RL = NT / NV;  // threads per channel vector
  constexpr int SBF = LDSF / (NT * VE);
  static_assert(NT % NV == 0 && VE % 4 == 0 && SBF >= 1, "one slot of the tile fits in lds");
  constexpr int SB = SBF < J ? SBF : J;
  const int t = threadIdx.x;
#pragma unroll
  for (int k0 = 0; k0 < J; k0 += SB) {
    const int kn = J - k0 < SB ? J - k0 : SB;
    __syncthreads();  // lds may still be read (the staged tile, or the previous slots)
#pragma unroll
    for (int kk = 0; kk < SB; ++kk)
      if (kk < kn)
#pragma unroll
        for (int j = 0; j < VE; j += 4)
          *(f4*)&lds[(kk * NT + t) * VE + j] =
              f4{acc[k0 + kk][j], acc[k0 + kk][j + 1], acc[k0 + kk][j + 2], acc[k0 + kk][j + 3]};
    __syncthreads();
    for (int item = t; item < kn * NV * VE; item += NT) {
      const int kk = item / (NV * VE), e = item - kk * (NV * VE);
      const float* col = lds + kk * NT * VE + e;  // thread l * NV + v holds (v * VE + j) at l * NV * VE
      float s = 0.f;
#pragma unroll 8
      for (int l = 0; l < RL; ++l) s += col[l * NV * VE];
      const int c = n0 + e;
      if (c < g.cp) g.part[((int64_t)(k0 + kk) * g.cp + c) * g.PM + tm] = s;
    }
  }
}

}  // namespace sscn
