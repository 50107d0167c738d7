// Block-level pieces of the ground-row chain of the backward pass (Section 2.3:
// the ground state stands for every inactive site, so its gradient is a sum),
// callable from their own kernels or as extra workgroups of another launch.
#pragma once

#include "common.h"
#include "kernels.h"

namespace sscn {

// Final pass of the bias / ground-row sums of one convolution for output
// channel c, by one workgroup of any multiple of 64 threads (at most 256): each
// wave sums its share of each slot's partials (lane-strided), reduces with a
// butterfly, and the wave sums are added in a fixed order (the same every run
// for a given workgroup size).  Thread 0 finishes:
//   with a pooling layer above, row 0 of delta is
//     z0 = f'(Y_below[0][c]) * (dY[0][c] + slot 0), written to delta[0][c]
//     (dY[0][c] read, or passed in as dy0 when inline_dy0);
//   without one, z0 = delta[0][c] as stored;
//   db[c] = slot 1 + z0,  D0[f][c] = slot 2+f + z0  (row 0 reads the ground row
//   at every window position), for c < c_out.
template <typename T, int AC>
__device__ inline void ground_final_block(const GroundArgs& g, int c, bool inline_dy0 = false, float dy0 = 0.f) {
  __shared__ float wsum[4][2 + AC];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const bool pool = g.B1 > 0;
  float tot[2 + AC];
#pragma unroll
  for (int k = 0; k < 2 + AC; ++k) tot[k] = 0.f;
  const float* pc = g.part + (int64_t)c * g.PM;
  const int64_t slot = (int64_t)g.cp * g.PM;
  int B1 = g.B1, B2 = g.B2;
  if (g.route_bm > 0) {  // one partial per row tile actually present
    const int tiles = (*g.n_pool + g.route_bm - 1) / g.route_bm;
    B1 = min(B1, tiles);
    B2 = min(B2, tiles);
  }
  const int npm = max(B1, B2);
#pragma unroll 2
  for (int p = threadIdx.x; p < npm; p += blockDim.x) {
    if (p < B1) tot[0] += pc[p];
    if (p < B2) {
#pragma unroll
      for (int k = 1; k < 2 + AC; ++k) tot[k] += pc[k * slot + p];
    }
  }
#pragma unroll
  for (int k = 0; k < 2 + AC; ++k) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) tot[k] += __shfl_xor(tot[k], off);
    if (lane == 0) wsum[w][k] = tot[k];
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
#pragma unroll
  for (int k = 0; k < 2 + AC; ++k) {
    float s = wsum[0][k];
    for (int q = 1; q < nw; ++q) s += wsum[q][k];
    tot[k] = s;
  }
  T* dZ = (T*)g.dZ;
  float z0;
  if (pool) {
    const float dy = inline_dy0 ? dy0 : Elem<T>::to_f32(((const T*)g.dY)[c]);
    const T g0 = Elem<T>::from_f32((tot[0] + dy) *
                                   act_factor(Elem<T>::to_f32(((const T*)g.Y_below)[c]), g.slope));
    dZ[c] = g0;
    z0 = Elem<T>::to_f32(g0);
  } else {
    z0 = Elem<T>::to_f32(dZ[c]);
  }
  if (c >= g.c_out) return;
  g.db[c] = tot[1] + z0;
#pragma unroll
  for (int k = 0; k < AC; ++k) g.D0[(int64_t)k * g.c_out + c] = tot[2 + k] + z0;
}

// Row 0 of the gradient below for input channel c (see Row0Args), by one
// workgroup of any power-of-two size up to 256 (fixed-order tree reduction).
// Thread 0 also returns the stored value (as float; 0 when c >= cp_in).
template <typename T>
__device__ inline float row0_dx_block(const Row0Args& r, int c) {
  __shared__ float red[256];
  float s = 0.f;
  if (c < r.c_in) {
    const T* W = (const T*)r.W;
    const int len = r.A * r.c_out;
    for (int t = threadIdx.x; t < len; t += blockDim.x) {
      const int f = t / r.c_out, n = t - f * r.c_out;
      s += Elem<T>::to_f32(W[((int64_t)f * r.c_in + c) * r.c_out + n]) * r.D0[t];
    }
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int off = blockDim.x >> 1; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off) red[threadIdx.x] += red[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0 && c < r.cp_in) {
    float v = red[0];
    if (r.Y_below) v *= act_factor(Elem<T>::to_f32(((const T*)r.Y_below)[c]), r.slope);
    const T t = Elem<T>::from_f32(v);
    ((T*)r.grad_in)[c] = t;
    return Elem<T>::to_f32(t);
  }
  return 0.f;
}

// Runs the extra task when this workgroup is one of the last x.blocks of the
// grid; returns whether it did (the caller then returns at once).  The other
// workgroups see a grid of gridDim.x - x.blocks.
template <typename T>
__device__ inline bool run_extra(const ExtraTask& x) {
  if (x.kind == 0) return false;
  const int first = (int)gridDim.x - x.blocks;
  if ((int)blockIdx.x < first) return false;
  const int i = (int)blockIdx.x - first;
  if (x.kind == 1 || x.kind == 3) {
    const bool in0 = x.kind == 3;
    const float dy0 = in0 ? row0_dx_block<T>(x.r, i) : 0.f;
    switch (x.AC) {
      case 0: ground_final_block<T, 0>(x.g, i, in0, dy0); break;
      case 1: ground_final_block<T, 1>(x.g, i, in0, dy0); break;
      case 4: ground_final_block<T, 4>(x.g, i, in0, dy0); break;
      default: ground_final_block<T, 9>(x.g, i, in0, dy0); break;
    }
  } else {
    row0_dx_block<T>(x.r, i);
  }
  return true;
}

__device__ inline int own_grid(const ExtraTask& x) { return (int)gridDim.x - (x.kind ? x.blocks : 0); }

}  // namespace sscn
