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

enum : int32_t { ERRBIT_RANGE = 1, ERRBIT_DUP = 2, ERRBIT_ORDER = 4, ERRBIT_LABEL = 8 };

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

// ---------------------------------------------------------------------------
// dropout masks (Section 2.1)
//
// Philox4x32-10, the counter-based generator of Salmon, Moraes, Dror and Shaw
// (SC 2011), from its definition: ten rounds over a four-word counter under a
// two-word key; a round takes the 64-bit products M0*c0 and M1*c2 and maps
// (c0, c1, c2, c3) to (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1,
// lo(M0 c0)); the key advances by two Weyl constants between rounds.

struct Philox4 {
  uint32_t w[4];
};

__host__ __device__ inline Philox4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0,
                                                 uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
    c1 = (uint32_t)p1;
    c3 = (uint32_t)p0;
    c0 = n0;
    c2 = n2;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return Philox4{{c0, c1, c2, c3}};
}

// Inverted dropout of one level: element (row key q, channel c) is kept, and
// multiplied by scale = 1/(1 - p), when word c % 4 of
// philox4x32_10(q, c / 4, level, 0; seed_lo, seed_hi) is >= thr = floor(p 2^32);
// otherwise it becomes 0.  Row keys: the packed site keys (b*S + y)*S + x of
// rows 1.. of a layer (keys[r - 1] for row r; row 0, the ground state, is never
// dropped), or the sample index for the softmax layer's input (keys null).
struct DropArgs {
  const int32_t* keys;
  uint32_t thr;
  uint32_t level;
  uint32_t seed_lo, seed_hi;
  float scale;
  int32_t on;  // 0: no dropout
};

// Factors of the four channels 4*c4 .. 4*c4 + 3 of row key q.
__device__ inline void drop_factors4(const DropArgs& d, uint32_t q, uint32_t c4, float f[4]) {
  const Philox4 r = philox4x32_10(q, c4, d.level, 0u, d.seed_lo, d.seed_hi);
#pragma unroll
  for (int e = 0; e < 4; ++e) f[e] = r.w[e] >= d.thr ? d.scale : 0.f;
}

__device__ inline float drop_factor(const DropArgs& d, uint32_t q, int c) {
  const Philox4 r = philox4x32_10(q, (uint32_t)c >> 2, d.level, 0u, d.seed_lo, d.seed_hi);
  const int e = c & 3;  // selects, not a dynamically indexed array
  const uint32_t w = e == 0 ? r.w[0] : e == 1 ? r.w[1] : e == 2 ? r.w[2] : r.w[3];
  return w >= d.thr ? d.scale : 0.f;
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
  // composite window of layer s on the input grid: output (Y, X) is active iff
  // an input site lies in [rf_a Y, rf_a Y + rf_r - 1] x [rf_a X, rf_a X + rf_r - 1]
  int32_t rf_a[MAX_LAYERS];
  int32_t rf_r[MAX_LAYERS];
  int32_t* rules[MAX_LAYERS];    // layer s >= 1: [(cap_s+1) * A]
  int32_t* rules_t[MAX_LAYERS];  // layer s >= 1: conv [(cap_{s-1}+1) * A], pool [cap_{s-1}+1]
  // pooling layer s on a 2x2 convolution (null otherwise): [cap_s + 1] child
  // ground masks, bit 4 f + k set when window position k of the convolution
  // row at pooling position f reads an inactive location of layer s - 2
  uint16_t* gmask[MAX_LAYERS];
  int32_t* counts;               // [nlayers]
  int32_t* err;                  // this build's error word (zero on entry)
  int32_t* err_next;             // the next build's error word, cleared here
  uint64_t* bits0_next;          // the next build's input bitmap [batch_max * S0 * Wd0], cleared here
  int32_t batch_max;
  int32_t* perm;                 // [n] row of each caller site (or -1)
  int32_t* head_rows;            // [batch]
  const int32_t* coords;         // [n][3]
  int32_t n;
  const int32_t* sample_begin;   // [batch + 1] when the sites are grouped by sample (no insertion launch), else null
};

__host__ __device__ inline int64_t round_up(int64_t a, int64_t b) { return (a + b - 1) / b * b; }

}  // namespace sscn
