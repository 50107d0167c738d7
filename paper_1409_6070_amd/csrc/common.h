// Internal definitions shared by the HIP kernels and the host planner.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>
#include <stdint.h>

namespace sscn {

// ---------------------------------------------------------------------------
// element types

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct alignas(16) Vec16 {  // one 16-byte vector of storage elements
  uint32_t w[4];
};

template <typename T>
struct Elem;
template <>
struct Elem<float> {
  static constexpr int VE = 4;  // elements per 16-byte vector
  __device__ static inline float to_f32(float v) { return v; }
  __device__ static inline float from_f32(float v) { return v; }
};
template <>
struct Elem<__bf16> {
  static constexpr int VE = 8;
  __device__ static inline float to_f32(__bf16 v) { return (float)v; }
  // round to nearest even (the conversion the compiler emits for float -> __bf16)
  __device__ static inline __bf16 from_f32(float v) { return (__bf16)v; }
};

// ---------------------------------------------------------------------------
// device error latch bits

enum : int32_t { ERRBIT_RANGE = 1, ERRBIT_DUP = 2 };

// ---------------------------------------------------------------------------
// per-layer geometry of the occupancy bitmaps

constexpr int MAX_LAYERS = 27;  // DeepCNet 2*ell + 2, DeepCNiN 3*ell + 3 layers, ell <= 8

// Derivative of a hidden layer's rectifier, decided from its stored output y:
// ReLU (slope 0): 1 for y > 0, else 0 (so ReLU'(0) = 0); leaky rectifier
// (slope 1/3): 1 on the x >= 0 branch (sign bit of y clear), else the slope.
__device__ inline float act_factor(float y, float slope) {
  const bool pos = slope == 0.f ? (y > 0.f) : !__builtin_signbit(y);
  return pos ? 1.f : slope;
}

struct LayerBits {
  uint64_t* bits;    // [batch * S * Wd] row-aligned occupancy words
  int32_t* wpre;     // [batch * S * Wd] exclusive popcount prefix within the sample
  int32_t* scount;   // [batch] active sites per sample
  int32_t* soff;     // [batch] exclusive prefix of scount over samples
  int32_t* sites;    // [cap] packed keys of rows 1..n
  int32_t S;
  int32_t Wd;        // 64-bit words per row
};

struct RulebookArgs {
  int32_t nlayers;
  int32_t batch;
  LayerBits L[MAX_LAYERS];
  int32_t kind[MAX_LAYERS];  // per layer s >= 1: 1 conv (F = 3, 2 or 1), 2 pool
  int32_t F[MAX_LAYERS];
  int32_t* rules[MAX_LAYERS];    // layer s >= 1: [(cap_s+1) * A]
  int32_t* rules_t[MAX_LAYERS];  // layer s >= 1: conv [(cap_{s-1}+1) * A], pool [cap_{s-1}+1]
  int32_t* counts;               // [nlayers]
  int32_t* err;
  int32_t* perm;                 // [n] row of each caller site (or -1)
  int32_t* head_rows;            // [batch]
  const int32_t* coords;         // [n][3]
  int32_t n;
};

__host__ __device__ inline int64_t round_up(int64_t a, int64_t b) { return (a + b - 1) / b * b; }

}  // namespace sscn
