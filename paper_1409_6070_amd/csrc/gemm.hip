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
//  * weight grad  dW = G^T delta, split over sites (for the softmax layer one
//                 extra A row of ones also gives db = sum delta).
//
// bf16: v_mfma_f32_16x16x32_bf16 (one per 32-wide k block);
// fp32: v_mfma_f32_16x16x4f32 (four per 16-wide k block).  Accumulation is
// always fp32.

#include "common.h"
#include "epilogue.h"
#include "pool_route.h"
#include "ground_tasks.h"
#include "kernels.h"

#include <hip/hip_ext.h>

#include <type_traits>

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

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Tile configuration: WM x WN waves, each computing TM x TN 16x16 MFMA tiles;
// K advances in slabs of 128 bytes per row (64 bf16 / 32 fp32 elements).
template <typename T, int WM_, int WN_, int TM_, int TN_>
struct GCfg {
  static constexpr int WM = WM_, WN = WN_, TM = TM_, TN = TN_;
  static constexpr int NT = 64 * WM * WN;
  static constexpr int BM = WM * TM * 16, BN = WN * TN * 16;
  static constexpr int VE = Elem<T>::VE;
  static constexpr int KB = MfmaCore<T>::KB;
  static constexpr int BK = 2 * KB;
  static constexpr int KV = BK / VE;       // 16-byte vectors per row and slab
  static constexpr int LDK = BK + VE;      // LDS row pitch (elements), padded against bank conflicts
  static constexpr int AV = BM * KV / NT;  // A vectors per thread and slab
  static constexpr int BV = BN * KV / NT;
  static_assert(AV * NT == BM * KV && BV * NT == BN * KV, "tile must split evenly over the threads");
};

constexpr int AMAX = 9;  // largest window (3x3)

// the four tile shapes (index = GemmArgs::cfg)
template <typename T> using C128x128 = GCfg<T, 2, 2, 4, 4>;
template <typename T> using C128x64 = GCfg<T, 4, 1, 2, 4>;
template <typename T> using C64x64 = GCfg<T, 2, 2, 2, 2>;
template <typename T> using C32x64 = GCfg<T, 2, 2, 1, 2>;

template <class C>
constexpr bool stages_tile() {
  return C::BM * (C::BN + C::VE) <= (C::BM + C::BN) * C::LDK;
}

bool gemm_routes(bool bf16, int cfg) {
  if (cfg == GEMM_DIRECT) return bf16;
  switch (cfg) {
    case 0: return bf16 ? stages_tile<C128x128<__bf16>>() : stages_tile<C128x128<float>>();
    case 1: return bf16 ? stages_tile<C128x64<__bf16>>() : stages_tile<C128x64<float>>();
    case 2: return bf16 ? stages_tile<C64x64<__bf16>>() : stages_tile<C64x64<float>>();
    default: return bf16 ? stages_tile<C32x64<__bf16>>() : stages_tile<C32x64<float>>();
  }
}

int gemm_bm(bool bf16, int cfg) { return cfg == GEMM_DIRECT ? DIRECT_BM : gemm_tile(bf16, cfg).BM; }

GemmTile gemm_tile(bool bf16, int cfg) {
  const int BK = bf16 ? 64 : 32;
  switch (cfg) {
    case 0: return GemmTile{128, 128, BK};
    case 1: return GemmTile{128, 64, BK};
    case 2: return GemmTile{64, 64, BK};
    default: return GemmTile{32, 64, BK};
  }
}

// acc[i][j] += A_tile(wave rows i) * B_tile(wave cols j) over one slab in LDS
template <typename T, class C>
__device__ inline void mma_slab(const T* As, const T* Bs, f32x4 (&acc)[C::TM][C::TN], int wm, int wn, int lane) {
  const int r16 = lane & 15, g = lane >> 4;
#pragma unroll
  for (int kb = 0; kb < C::BK; kb += C::KB) {
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
      for (int j = 0; j < C::TN; ++j)
        MfmaCore<T>::step(As + (wm * C::TM * 16 + i * 16 + r16) * C::LDK + kb + g * C::VE,
                          Bs + (wn * C::TN * 16 + j * 16 + r16) * C::LDK + kb + g * C::VE, acc[i][j]);
  }
}

// acc += A_tile * B_tile over one slab held in LDS unpadded and swizzled (the
// bf16 pipeline below): row r's 16-byte chunk c sits in slot c ^ ((r / 2) % 8)
// of its 128-byte row, so the sixteen rows an MFMA operand read touches cover
// all 64 banks once.
template <class C>
__device__ inline void mma_slab_sw(const __bf16* As, const __bf16* Bs, f32x4 (&acc)[C::TM][C::TN], int wm, int wn,
                                   int lane) {
  const int r16 = lane & 15, g = lane >> 4;
#pragma unroll
  for (int kb = 0; kb < C::BK; kb += C::KB) {
    const int chunk = kb / 8 + g;
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
      for (int j = 0; j < C::TN; ++j) {
        const int ra = wm * C::TM * 16 + i * 16 + r16, rb = wn * C::TN * 16 + j * 16 + r16;
        MfmaCore<__bf16>::step(As + ra * C::BK + ((chunk ^ ((ra >> 1) & 7)) * 8),
                               Bs + rb * C::BK + ((chunk ^ ((rb >> 1) & 7)) * 8), acc[i][j]);
      }
  }
}

// s_waitcnt vmcnt(n) lgkmcnt(0), n a compile-time constant: the LDS reads of
// the previous slab are done before its stage is refilled
template <int N>
__device__ inline void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));  // lgkmcnt(0) too
}

// One 16-byte load per lane from a buffer straight into LDS: lane l's bytes
// land at LDS byte address lds + 16 l (lds uniform over the wave). An offset
// at or past the buffer's size reads zero. The compiler does not see this
// load, so the caller waits for it with wait_vmcnt; its own waits only grow
// stricter with loads it does not know of. No memory clobber: the caller
// orders the load against the LDS reads of the same stage with compiler
// fences around its barriers.
__device__ inline void dma16(u32x4 rsrc, uint32_t lds, uint32_t off) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %1, %2, 0 offen lds" ::"s"(lds),
      "v"(off), "s"(rsrc)
      : "m0");
}

// The same for 4 bytes per lane: lane l's dword lands at lds + 4 l.
__device__ inline void dma4(u32x4 rsrc, uint32_t lds, uint32_t off) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "buffer_load_dword %1, %2, 0 offen lds" ::"s"(lds),
      "v"(off), "s"(rsrc)
      : "m0");
}

// raw buffer descriptor: base, no stride, size in bytes
__device__ inline u32x4 buffer_rsrc(const void* base, uint32_t bytes) {
  const uint64_t b = (uint64_t)base;
  return u32x4{(uint32_t)b, (uint32_t)(b >> 32) & 0xffffu, bytes, 0x00020000u};
}

__device__ inline uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// q = k / d for 0 <= k < 2^20, 1 <= d < 2^16: float estimate, then exact correction.
__device__ inline int div_small(int k, int d, float rcp) {
  int q = (int)((float)k * rcp);
  q += (q + 1) * d <= k ? 1 : 0;
  q -= q * d > k ? 1 : 0;
  return q;
}

// Routing inputs of the items a thread takes in store_staged (AC >= 0 and at
// most two items per thread), all loaded before the first item is routed: one
// memory round trip for the thread's items, not one each.
template <typename T, class C, int AC>
struct StagedRoute {
  static constexpr int NV = C::BN / C::VE;
  static constexpr int IPT = (C::BM * NV + C::NT - 1) / C::NT;  // items per thread
  static constexpr bool ON = AC >= 0 && IPT <= 2;
  RouteIn<T, AC < 0 ? 0 : AC> q[ON ? IPT : 1];
  __device__ inline void load(const GemmArgs& a, int m0, int n0, int rows) {
    if constexpr (ON) {
#pragma unroll
      for (int i = 0; i < IPT; ++i) {
        const int v = threadIdx.x + i * C::NT;
        const int r = v / NV, m = m0 + r, n = n0 + (v - r * NV) * C::VE;
        if (v < C::BM * NV && m >= 1 && m < rows && n < a.out_cols)
          route_load_window<T, AC < 0 ? 0 : AC>(a.pr, m, n, q[i]);
      }
    }
  }
};

// Stores of an output tile staged in LDS (Cs, pitch CS), 16 bytes at a time.
// AC >= 0: the pooling backward of every row m >= 1 as well, and the tile's
// slot partial sums as partial tm (lds: the staging buffer, reused).
template <typename T, class C, int CS, int AC>
__device__ inline void store_staged(const GemmArgs& a, const T* Cs, int m0, int n0, int tm, int rows, float* lds) {
  constexpr int VE = C::VE, BM = C::BM, BN = C::BN, NT = C::NT, NV = BN / VE;
  constexpr int J = AC >= 0 ? 2 + AC : 1;
  static_assert(NT % NV == 0, "each thread keeps one channel vector");
  float acc[J][VE];
  if constexpr (AC >= 0) {
#pragma unroll
    for (int k = 0; k < J; ++k)
#pragma unroll
      for (int e = 0; e < VE; ++e) acc[k][e] = 0.f;
  }
  if constexpr (StagedRoute<T, C, AC>::ON) {
    StagedRoute<T, C, AC> pre;
    pre.load(a, m0, n0, rows);
#pragma unroll
    for (int i = 0; i < StagedRoute<T, C, AC>::IPT; ++i) {
      const int v = threadIdx.x + i * NT;
      const int r = v / NV, nv = v - r * NV;
      const int m = m0 + r, n = n0 + nv * VE;
      if (v < BM * NV && m < rows && n < a.out_cols) {
        const u32x4 o = *(const u32x4*)(Cs + r * CS + nv * VE);
        *(u32x4*)((T*)a.out + (int64_t)m * a.out_stride + n) = o;
        if (m >= 1) {
          route_load_children<T, AC>(a.pr, n, pre.q[i]);
          route_apply<T, AC>(a.pr, n, pre.q[i], (const T*)&o, acc);
        }
      }
    }
  } else {
    for (int v = threadIdx.x; v < BM * NV; v += NT) {
      const int r = v / NV, nv = v - r * NV;
      const int m = m0 + r, n = n0 + nv * VE;
      if (m < rows && n < a.out_cols) {
        const u32x4 o = *(const u32x4*)(Cs + r * CS + nv * VE);
        *(u32x4*)((T*)a.out + (int64_t)m * a.out_stride + n) = o;
        if constexpr (AC >= 0)
          if (m >= 1) pool_route_item<T, AC>(a.pr, m, n, (const T*)&o, acc);
      }
    }
  }
  if constexpr (AC >= 0) tile_slot_sums<VE, J, NT, NV, (BM + BN) * C::LDK * (int)sizeof(T) / 4>(acc, lds, a.pr, n0, tm);
}

// Pooling forward in the epilogue (GemmArgs::pool_fwd): the staged tile's
// rows are the slots 4 p + f of pooling windows p (m0 is a multiple of 4).
// Every slot's convolution row Cr is stored (row 0 from slot 0 only: the
// ground value), then each window's first maximum over its four slots, per
// channel, goes to the pooling layer with its position.
template <typename T, class C, int CS>
__device__ inline void store_pooled(const GemmArgs& a, const T* Cs, const int32_t* Cr, int m0, int n0, int rows) {
  constexpr int VE = C::VE, BM = C::BM, BN = C::BN, NT = C::NT, NV = BN / VE;
  typedef typename ArgPack<VE>::W AW;
  static_assert(BM % 4 == 0, "whole windows per tile");
  for (int v = threadIdx.x; v < BM * NV; v += NT) {
    const int r = v / NV, nv = v - r * NV;
    const int m = m0 + r, n = n0 + nv * VE;
    const int row = Cr[r];
    if (m < rows && n < a.out_cols && (row > 0 || m == 0))
      *(u32x4*)((T*)a.out + (int64_t)row * a.out_stride + n) = *(const u32x4*)(Cs + r * CS + nv * VE);
  }
  for (int v = threadIdx.x; v < (BM / 4) * NV; v += NT) {
    const int pr = v / NV, nv = v - pr * NV;
    const int m = m0 + 4 * pr, n = n0 + nv * VE;
    if (m >= rows || n >= a.out_cols) continue;
    // running first maximum over the four slots (one staged vector at a time)
    u32x4 out = *(const u32x4*)(Cs + (4 * pr) * CS + nv * VE);
    AW am = 0;
#pragma unroll
    for (int f = 1; f < 4; ++f) {
      const u32x4 in = *(const u32x4*)(Cs + (4 * pr + f) * CS + nv * VE);
#pragma unroll
      for (int j = 0; j < VE; ++j) {
        const bool gt = Elem<T>::to_f32(((const T*)&in)[j]) > Elem<T>::to_f32(((const T*)&out)[j]);
        if (gt) {
          ((T*)&out)[j] = ((const T*)&in)[j];
          am = (am & ~((AW)0xff << (8 * j))) | ((AW)f << (8 * j));
        }
      }
    }
    const int64_t p = m / 4;
    *(u32x4*)((T*)a.pool_out + p * a.pool_stride + n) = out;
    *(AW*)(a.pool_argmax + p * a.pool_stride + n) = am;
  }
}

// Implicit-gather GEMM.  Per tile: the tile's window rows go to LDS once; the
// K slabs stream through a ring of LDS stages filled by buffer loads with an
// LDS destination (bf16; float32 prefetches the next slab into registers);
// the output tile is staged in LDS for 16-byte stores.
// With ksplit > 1 each workgroup covers one K range and writes fp32 partial
// sums, reduced (with the epilogue) by k_gemm_splitk_reduce.
template <typename T, class C, int RAC>
__global__ void __launch_bounds__(C::NT) k_gemm_gather(GemmArgs a) {
  constexpr int VE = C::VE, BK = C::BK, KV = C::KV, LDK = C::LDK, BM = C::BM, BN = C::BN, NT = C::NT;
  constexpr int SMEM = (BM + BN) * LDK;
  constexpr int CS = BN + VE;  // staging pitch
  constexpr bool STAGE = stages_tile<C>();
  static_assert(STAGE == (BM * CS <= SMEM), "staging fits");
  constexpr bool POOL = RAC == POOL_FWD_MODE;
  // bf16: the operands go from memory straight into LDS (buffer loads with an
  // LDS destination; an offset past the buffer reads zero), NST slabs in LDS,
  // NST - 1 of them in flight while one is multiplied, one barrier per slab.
  // Two stages where three would cost occupancy (the 128x128 tile; the pooled
  // forward, which then fits three workgroups per compute unit and its
  // launches one round of workgroups) or measured slower (the routed tiles,
  // whose epilogue holds more registers).
  constexpr bool DMA = sizeof(T) == 2;
  constexpr int NST = (BM + BN >= 256 || RAC >= 0 || POOL) ? 2 : 3;
  constexpr int STG = (BM + BN) * BK;          // elements per stage
  constexpr int LPS = C::AV + C::BV;           // loads per thread and slab
  constexpr int SMEM_ALL = DMA ? (NST * STG > SMEM ? NST * STG : SMEM) : SMEM;
  __shared__ __attribute__((aligned(16))) T smem[SMEM_ALL];
  extern __shared__ int32_t Rs[];  // [BM * A] window entries, sized at launch
  __shared__ int32_t Cr[POOL ? BM : 1];  // pooling forward: the convolution row of each slot
  T* As = smem;
  T* Bs = smem + BM * LDK;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / C::WN, wn = wave % C::WN;
  if (run_extra<T>(a.x)) return;
  const int rows = (a.rows_dev ? (*a.rows_dev + a.rows_add) : a.rows_host) * (POOL ? 4 : 1);
  const int span = rows - a.row_begin;
  if (span <= 0) return;
  const int tiles_m = (span + BM - 1) / BM;
  const int tiles_n = a.Npad / BN;
  const int kslabs = a.Kpad / BK;
  const int kper = (kslabs + a.ksplit - 1) / a.ksplit * BK;
  const int ntiles = tiles_m * tiles_n * a.ksplit;
  const T* src = (const T*)a.src;
  const T* Bt = (const T*)a.Bt;
  const int A = a.A;

  const int grid = own_grid(a.x);
  for (int tile = blockIdx.x; tile < ntiles; tile += grid) {
    const int tn = tile % tiles_n;
    const int t2 = tile / tiles_n;
    const int tm = t2 % tiles_m;
    const int ks = t2 / tiles_m;
    const int m0 = a.row_begin + tm * BM, n0 = tn * BN;
    const int kbeg = ks * kper;
    const int kend = min(a.Kpad, kbeg + kper);

    if (tid < BM) {  // the tile's window rows: one row per thread, all loads issued before any store
      const int m = m0 + tid;
      const bool live = m < rows;
      int row = m;  // the output row (pooling forward: the slot's convolution row)
      if constexpr (POOL) {
        const int pr = a.pslot[live ? m : 0];
        row = live ? pr : 0;
        Cr[tid] = row;
      }
      int v[AMAX];
      if (a.rmap) {  // rows past the count read row 0's window and discard it
        const int32_t* rp = a.rmap + (int64_t)(live ? row : 0) * A;
#pragma unroll
        for (int f = 0; f < AMAX; ++f) v[f] = rp[f < A ? f : 0];
      } else {
#pragma unroll
        for (int f = 0; f < AMAX; ++f) v[f] = f == 0 ? row : -1;
      }
#pragma unroll
      for (int f = 0; f < AMAX; ++f)
        if (f < A) Rs[tid * A + f] = live ? v[f] : -1;
    }
    __syncthreads();

    f32x4 acc[C::TM][C::TN];
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
      for (int j = 0; j < C::TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const float rcp_cseg = 1.f / (float)a.cseg;
    if constexpr (DMA) {
      // A: one 16-byte slot per load (row v / 8, slot v % 8 holding chunk
      // (v % 8) ^ ((row / 2) % 8)); rows without a window entry and k past K read zero
      const u32x4 rsA = buffer_rsrc(src, GATHER_SRC_BYTES);
      const u32x4 rsB = buffer_rsrc(Bt, (uint32_t)a.Npad * (uint32_t)a.Kpad * 2u);
      const int wave_u = __builtin_amdgcn_readfirstlane(wave);  // in a scalar register
      const uint32_t lds0 = lds_addr(smem);
      auto issue = [&](int k0, int st) {
        const uint32_t la = lds0 + (uint32_t)(st * STG) * 2u, lb = la + BM * BK * 2;
        uint32_t off[C::AV];
#pragma unroll
        for (int j = 0; j < C::AV; ++j) {  // every window row read before the first load goes out
          const int v = tid + j * NT;
          const int r = v >> 3, c = (v & 7) ^ ((r >> 1) & 7);
          const int k = k0 + c * 8;
          const bool in_k = k < a.K;
          const int f = div_small(k, a.cseg, rcp_cseg);
          const int srow = Rs[r * A + (in_k ? f : 0)];
          off[j] = in_k && srow >= 0 ? (uint32_t)(srow * a.src_stride + (k - f * a.cseg)) * 2u : GATHER_SRC_BYTES;
        }
#pragma unroll
        for (int j = 0; j < C::AV; ++j) dma16(rsA, la + (uint32_t)(wave_u * 64 + j * NT) * 16u, off[j]);
#pragma unroll
        for (int j = 0; j < C::BV; ++j) {
          const int v = tid + j * NT;
          const int r = v >> 3, c = (v & 7) ^ ((r >> 1) & 7);
          dma16(rsB, lb + (uint32_t)(wave_u * 64 + j * NT) * 16u, (uint32_t)((n0 + r) * a.Kpad + k0 + c * 8) * 2u);
        }
      };
      const int nsl = (kend - kbeg) / BK;
#pragma unroll
      for (int p = 0; p < NST - 1; ++p)
        if (p < nsl) issue(kbeg + p * BK, p);
      for (int s = 0; s < nsl; ++s) {
        // this wave's loads of slab s have landed once at most those of the
        // slabs after it are outstanding; the barrier makes it every wave's
        asm volatile("" ::: "memory");
        if constexpr (NST == 3) {
          if (s + 1 < nsl) wait_vmcnt<LPS>(); else wait_vmcnt<0>();
        } else {
          wait_vmcnt<0>();
        }
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        if (s + NST - 1 < nsl) issue(kbeg + (s + NST - 1) * BK, (s + NST - 1) % NST);
        mma_slab_sw<C>(smem + (s % NST) * STG, smem + (s % NST) * STG + BM * BK, acc, wm, wn, lane);
      }
      asm volatile("" ::: "memory");
      __syncthreads();  // every wave done with the slabs before the epilogue reuses the memory
    } else {
      u32x4 ra[C::AV], rb[C::BV];
      auto load = [&](int k0) {
        int srow[C::AV], col[C::AV];
#pragma unroll
        for (int j = 0; j < C::AV; ++j) {  // window row and channel of each vector, then all loads at once
          const int v = tid + j * NT;
          const int r = v / KV, kv = v - r * KV;
          const int k = k0 + kv * VE;
          const bool in_k = k < a.K;
          const int f = in_k ? div_small(k, a.cseg, rcp_cseg) : 0;
          srow[j] = in_k ? Rs[r * A + f] : -1;
          col[j] = in_k ? k - f * a.cseg : 0;
        }
#pragma unroll
        for (int j = 0; j < C::AV; ++j) {
          const u32x4 val = *(const u32x4*)(src + (int64_t)max(srow[j], 0) * a.src_stride + col[j]);
          ra[j] = srow[j] >= 0 ? val : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int j = 0; j < C::BV; ++j) {
          const int v = tid + j * NT;
          const int r = v / KV, kv = v - r * KV;
          rb[j] = *(const u32x4*)(Bt + (int64_t)(n0 + r) * a.Kpad + k0 + kv * VE);
        }
      };
      if (kbeg < kend) load(kbeg);
      for (int k0 = kbeg; k0 < kend; k0 += BK) {
#pragma unroll
        for (int j = 0; j < C::AV; ++j) {
          const int v = tid + j * NT;
          const int r = v / KV, kv = v - r * KV;
          *(u32x4*)(As + r * LDK + kv * VE) = ra[j];
        }
#pragma unroll
        for (int j = 0; j < C::BV; ++j) {
          const int v = tid + j * NT;
          const int r = v / KV, kv = v - r * KV;
          *(u32x4*)(Bs + r * LDK + kv * VE) = rb[j];
        }
        __syncthreads();
        if (k0 + BK < kend) load(k0 + BK);
        mma_slab<T, C>(As, Bs, acc, wm, wn, lane);
        __syncthreads();
      }
    }

    const int g = lane >> 4, c16 = lane & 15;
    float bias[C::TN];
#pragma unroll
    for (int j = 0; j < C::TN; ++j) {
      const int n = n0 + wn * C::TN * 16 + j * 16 + c16;
      bias[j] = (a.bias && n < a.N) ? a.bias[n] : 0.f;
    }
    if (a.ksplit > 1) {
      float* part = a.part + (int64_t)ks * a.part_rows * a.Npad;
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j) {
          const int n = n0 + wn * C::TN * 16 + j * 16 + c16;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int m = m0 + wm * C::TM * 16 + i * 16 + g * 4 + r;
            if (m < rows) part[(int64_t)m * a.Npad + n] = acc[i][j][r];
          }
        }
    } else if (STAGE && epi_stores_T(a.epi)) {
      T* Cs = smem;
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j) {
          const int nl = wn * C::TN * 16 + j * 16 + c16;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int ml = wm * C::TM * 16 + i * 16 + g * 4 + r;
            float v = epi_value<T>(a, acc[i][j][r], bias[j]);
            if constexpr (RAC == MASK_MODE)  // the rectifier derivative of the layer below,
              if (m0 + ml < rows && n0 + nl < a.out_cols)  // before the one rounding to storage
                v *= act_factor(
                    Elem<T>::to_f32(((const T*)a.mask)[(int64_t)(m0 + ml) * a.mask_stride + n0 + nl]), a.slope);
            Cs[ml * CS + nl] = Elem<T>::from_f32(v);
          }
        }
      __syncthreads();
      if constexpr (POOL)
        store_pooled<T, C, CS>(a, Cs, Cr, m0, n0, rows);
      else
        store_staged<T, C, CS, RAC>(a, Cs, m0, n0, tm, rows, (float*)smem);
    } else {
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j) {
          const int n = n0 + wn * C::TN * 16 + j * 16 + c16;
          if (n >= a.out_cols) continue;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int m = m0 + wm * C::TM * 16 + i * 16 + g * 4 + r;
            if (m < rows) store_out<T>(a, m, n, epi_value<T>(a, acc[i][j][r], bias[j]));
          }
        }
    }
    __syncthreads();
  }
}

// Sum of the split-K partials plus the epilogue: four consecutive columns per
// thread, one 16-byte partial load per split (the partials are Npad wide).
template <typename T>
__global__ void __launch_bounds__(256) k_gemm_splitk_reduce(GemmArgs a) {
  const int rows = a.rows_dev ? (*a.rows_dev + a.rows_add) : a.rows_host;
  const int64_t span = rows - a.row_begin;
  if (span <= 0) return;
  const int quads = (a.out_cols + 3) / 4;
  const int64_t total = span * quads;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t m = a.row_begin + t / quads;
    const int n = (int)(t % quads) * 4;
    f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (int ks = 0; ks < a.ksplit; ++ks) s += *(const f32x4*)(a.part + ((int64_t)ks * a.part_rows + m) * a.Npad + n);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (n + e < a.out_cols) store_out<T>(a, m, n + e, epi_value<T>(a, s[e], (a.bias && n + e < a.N) ? a.bias[n + e] : 0.f));
  }
}

// Packs 4 consecutive-site values of one element into one LDS store.
template <typename T>
struct Quad;
template <>
struct Quad<__bf16> {
  typedef uint64_t W;
  __device__ static inline W pack(__bf16 a, __bf16 b, __bf16 c, __bf16 d) {
    return (uint64_t)__builtin_bit_cast(uint16_t, a) | ((uint64_t)__builtin_bit_cast(uint16_t, b) << 16) |
           ((uint64_t)__builtin_bit_cast(uint16_t, c) << 32) | ((uint64_t)__builtin_bit_cast(uint16_t, d) << 48);
  }
};
template <>
struct Quad<float> {
  typedef u32x4 W;
  __device__ static inline W pack(float a, float b, float c, float d) {
    return u32x4{__builtin_bit_cast(uint32_t, a), __builtin_bit_cast(uint32_t, b), __builtin_bit_cast(uint32_t, c),
                 __builtin_bit_cast(uint32_t, d)};
  }
};

// Site chunks actually used: slabs of BK sites per chunk as planned, at most
// the planned (capacity) chunk count, from the device-side row count.
__device__ inline int wgrad_chunks_dev(const WGradArgs& a, int rows, int BK) {
  const int want = (rows + a.slabs * BK - 1) / (a.slabs * BK);
  return max(1, min(a.nchunks, want));
}

// A tile's sums for one site chunk.  Several chunks: split-K partials stored
// as the MFMA result fragments, the layout the reduce reads: per chunk,
// 16 x 16 blocks (bm, bn) for bm < ceil(m_rows / 16), bn < ceil(c_out / 16)
// (blocks past the rows and columns read back are not stored), block
// bm * NB + bn holding 64 lanes x 4 floats, lane 16 g + c the rows 4 g .. 4 g + 3
// of column c; one 16-byte store per lane and block.  A single chunk: the sums
// are final and go to dW / db.
template <class C>
__device__ inline void store_wgrad_tile(const WGradArgs& a, const f32x4 (&acc)[C::TM][C::TN], int chunk, int nch,
                                        int m0, int n0, int wm, int wn, int lane, int m_rows, int m_gather) {
  const int g = lane >> 4, c16 = lane & 15;
  if (nch > 1) {
    const int MB = (m_rows + 15) / 16, NB = (a.c_out + 15) / 16;
    float* part = a.part + (int64_t)chunk * MB * NB * 256;
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
      for (int j = 0; j < C::TN; ++j) {
        const int bm = m0 / 16 + wm * C::TM + i, bn = n0 / 16 + wn * C::TN + j;
        if (bm < MB && bn < NB) *(f32x4*)(part + ((int64_t)(bm * NB + bn) * 64 + lane) * 4) = acc[i][j];
      }
    return;
  }
  // a lane's 4 rows 4 g .. 4 g + 3 of block i share one window position f
  // (cseg and the rows' first index are multiples of 4): one division per block
  const float rcp_cseg = 1.f / (float)a.cseg;
#pragma unroll
  for (int i = 0; i < C::TM; ++i) {
    const int mb = m0 + wm * C::TM * 16 + i * 16 + g * 4;
    const int f = div_small(mb, a.cseg, rcp_cseg), c = mb - f * a.cseg;
    int idx[4];
    bool wr[4], br[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      wr[r] = mb + r < m_gather && c + r < a.c_in;
      br[r] = mb + r == a.m_ones && a.db;
      idx[r] = (f * a.c_in + c + r) * a.c_out;
    }
#pragma unroll
    for (int j = 0; j < C::TN; ++j) {
      const int nn = n0 + wn * C::TN * 16 + j * 16 + c16;
      if (nn >= a.c_out) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (wr[r])
          a.dW[idx[r] + nn] = acc[i][j][r];
        else if (br[r])
          a.db[nn] = acc[i][j][r];
      }
    }
  }
}

// Weight-gradient GEMM, split over sites (the K dimension).  A^T and delta^T
// slabs are staged in LDS as [row of dW / col of dW][site]: each thread loads
// 16-byte vectors (VE consecutive channels) of 4 consecutive sites and stores
// them transposed, 4 sites per LDS write.  Loads of the next slab are issued
// before the current slab's MFMAs.
//
// One launch serves a group of layers: workgroup tile t belongs to the layer l
// with tile_beg[l] <= t < tile_beg[l + 1].
template <typename T, class C>
__global__ void __launch_bounds__(C::NT) k_wgrad(WGradGroup grp, ExtraTask x) {
  constexpr int VE = C::VE, BK = C::BK, LDK = C::LDK, BM = C::BM, BN = C::BN, NT = C::NT;
  constexpr int MV = BM / VE, NV = BN / VE;  // vectors across a slab row
  static_assert(MV * (BK / 4) == NT && NV * (BK / 4) <= NT, "one quad of sites per thread");
  typedef typename Quad<T>::W QW;
  __shared__ __attribute__((aligned(16))) T As[BM * LDK];  // [m][site]
  __shared__ __attribute__((aligned(16))) T Bs[BN * LDK];  // [n][site]

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / C::WN, wn = wave % C::WN;
  const T one = Elem<T>::from_f32(1.f), zero = Elem<T>::from_f32(0.f);
  // this thread's quad: sites 4*q .. 4*q+3 of a slab, vector mv / nv.  The quad
  // index runs fastest so that a wavefront's transposed LDS writes spread over
  // all banks (vector-fastest puts every vector of a quad on the same bank).
  constexpr int NQ = BK / 4;
  const int qa = tid % NQ, mv = tid / NQ;
  const int qb = tid % NQ, nvv = tid / NQ;
  const bool b_active = tid < NV * NQ;
  if (run_extra<T>(x)) return;

  for (int t = blockIdx.x; t < grp.tile_beg[grp.n]; t += own_grid(x)) {
    int l = 0;
    while (l + 1 < grp.n && t >= grp.tile_beg[l + 1]) ++l;
    const WGradArgs& a = grp.L[l];
    const int tile = t - grp.tile_beg[l];
    const int rows = a.rows_dev ? (*a.rows_dev + a.rows_add) : a.rows_host;
    const int tiles_m = a.Mpad / BM, tiles_n = a.Npad / BN;
    const int nch = wgrad_chunks_dev(a, rows, BK);
    const int per = ((rows + nch - 1) / nch + BK - 1) / BK * BK;
    const int m_gather = a.A * a.cseg;
    const int m_rows = a.m_ones >= 0 ? a.m_ones + 1 : m_gather;  // rows of dW / db that are read back
    const T* src = (const T*)a.src;
    const T* dsrc = (const T*)a.dsrc;
    const int tn = tile % tiles_n;
    const int tq = tile / tiles_n;
    const int tm = tq % tiles_m;
    const int chunk = tq / tiles_m;
    if (chunk >= nch) continue;  // fewer rows than the plan allowed for
    const int m0 = tm * BM, n0 = tn * BN;
    const int o_beg = chunk * per;
    const int o_end = min(rows, o_beg + per);
    f32x4 acc[C::TM][C::TN];
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
      for (int j = 0; j < C::TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    u32x4 ra[4], rb[4];
    const int m = m0 + mv * VE;
    const int f_of_m = m < m_gather ? m / a.cseg : 0;
    const int c_of_m = m < m_gather ? m - f_of_m * a.cseg : 0;
    const int n = n0 + nvv * VE;
    // source rows of this thread's 4 sites, fetched one slab ahead of their use
    int rnext[4];
    auto load_rows = [&](int ob) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int o = ob + 4 * qa + i;
        int r = -1;
        if (o < o_end && m < m_gather) r = a.rmap ? a.rmap[(int64_t)o * a.A + f_of_m] : o;
        rnext[i] = r;
      }
    };
    auto load = [&](int ob) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int o = ob + 4 * qa + i;
        u32x4 val = {0u, 0u, 0u, 0u};
        if (o < o_end) {
          if (m < m_gather) {
            val = *(const u32x4*)(src + (int64_t)rnext[i] * a.src_stride + c_of_m);
          } else {
            T* vv = (T*)&val;
#pragma unroll
            for (int j = 0; j < VE; ++j) vv[j] = (m + j == a.m_ones) ? one : zero;
          }
        }
        ra[i] = val;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int o = ob + 4 * qb + i;
        u32x4 val = {0u, 0u, 0u, 0u};
        if (b_active && o < o_end && n < a.dsrc_cols) val = *(const u32x4*)(dsrc + (int64_t)o * a.dsrc_stride + n);
        rb[i] = val;
      }
    };
    load_rows(o_beg);
    if (o_beg < o_end) {
      load(o_beg);
      load_rows(o_beg + BK);
    }
    for (int ob = o_beg; ob < o_end; ob += BK) {
#pragma unroll
      for (int j = 0; j < VE; ++j)
        *(QW*)(As + (mv * VE + j) * LDK + 4 * qa) =
            Quad<T>::pack(((const T*)&ra[0])[j], ((const T*)&ra[1])[j], ((const T*)&ra[2])[j], ((const T*)&ra[3])[j]);
      if (b_active) {
#pragma unroll
        for (int j = 0; j < VE; ++j)
          *(QW*)(Bs + (nvv * VE + j) * LDK + 4 * qb) = Quad<T>::pack(((const T*)&rb[0])[j], ((const T*)&rb[1])[j],
                                                                      ((const T*)&rb[2])[j], ((const T*)&rb[3])[j]);
      }
      __syncthreads();
      if (ob + BK < o_end) {
        load(ob + BK);
        load_rows(ob + 2 * BK);
      }
      mma_slab<T, C>(As, Bs, acc, wm, wn, lane);
      __syncthreads();
    }

    store_wgrad_tile<C>(a, acc, chunk, nch, m0, n0, wm, wn, lane, m_rows, m_gather);
  }
}

// Pair swizzle of an LDS row of sites for the transpose reads below: the
// 32-byte pair p of row r sits at pair slot p ^ swz(r).  A wavefront's read
// touches rows {0..3, 8..11} (+ 16, + 4, + 32) in each half, so the swizzle
// spreads each such set of eight rows over all 64 banks: 256-byte rows by
// (r % 4, r / 8 % 2), 128-byte rows (two per bank sweep) by (r / 2 % 2, r / 8 % 2).
template <int ROW_BYTES>
__device__ inline int site_row_swz(int r) {
  static_assert(ROW_BYTES == 256 || ROW_BYTES == 128, "row width");
  if constexpr (ROW_BYTES == 256)
    return (r & 3) | (((r >> 3) & 1) << 2);
  else
    return ((r >> 1) & 1) | (((r >> 3) & 1) << 1);
}

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

// 8 consecutive sites of one column as an MFMA operand (k = sites): two LDS
// transpose reads of 4 sites each.  Within each 16-lane group, lane q reads
// 4 columns (4 (q % 4) .. + 3) of site row q / 4 and receives column q of the
// group's 4 rows; `p` points at lane q's 4 columns of the group's first row.
template <int ROW>
__device__ inline bf16x8 tr_operand(const __bf16* p) {
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)lds_addr(p));
  const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)lds_addr(p + 4 * ROW));
  const s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

// acc += G_slab^T * delta_slab for one slab of BKS sites held as [site][column]
// (A: BM columns, B: BN columns, pair-swizzled rows).  ONES: this wave's rows
// hold the bias row m_loc, whose operand is 1 for each of the slab's first
// `valid` sites and 0 after.
template <class C, int BKS, bool ONES>
__device__ inline void mma_slab_tr(const __bf16* As, const __bf16* Bs, f32x4 (&acc)[C::TM][C::TN], int wm, int wn,
                                   int lane, int m_loc, int valid) {
  constexpr int BM = C::BM, BN = C::BN;
  const int g = lane >> 4, q = lane & 15;
  const int e4 = 4 * (q & 3);
#pragma unroll
  for (int kb = 0; kb < BKS; kb += C::KB) {
    const int row = kb + 8 * g + (q >> 2);
    const int ha = site_row_swz<BM * 2>(row), hb = site_row_swz<BN * 2>(row);
    bf16x8 bv[C::TN];
#pragma unroll
    for (int j = 0; j < C::TN; ++j) bv[j] = tr_operand<BN>(Bs + row * BN + (((wn * C::TN + j) ^ hb) << 4) + e4);
#pragma unroll
    for (int i = 0; i < C::TM; ++i) {
      bf16x8 av = tr_operand<BM>(As + row * BM + (((wm * C::TM + i) ^ ha) << 4) + e4);
      if constexpr (ONES) {
        if (wm * C::TM * 16 + i * 16 + q == m_loc) {
#pragma unroll
          for (int e = 0; e < 8; ++e) av[e] = (__bf16)(kb + 8 * g + e < valid ? 1.f : 0.f);
        }
      }
#pragma unroll
      for (int j = 0; j < C::TN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv[j], acc[i][j], 0, 0, 0);
    }
  }
}

// s_waitcnt vmcnt(BASE + STEP x steps) lgkmcnt(0), steps a run-time value in 0 .. 3
template <int BASE, int STEP>
__device__ inline void wait_vmcnt_steps(int steps) {
  switch (steps) {
    case 0: wait_vmcnt<BASE>(); break;
    case 1: wait_vmcnt<BASE + STEP>(); break;
    case 2: wait_vmcnt<BASE + 2 * STEP>(); break;
    default: wait_vmcnt<BASE + 3 * STEP>(); break;
  }
}

// Weight gradients, bf16: the tiles and site chunks of k_wgrad, but the operand
// slabs (BKS sites) go from memory straight into LDS as stored, one site per
// LDS row (buffer loads with an LDS destination; an offset past the buffer
// reads zero), and the MFMA operands are read across sites with the LDS
// transpose read.  NST stages: the loads of NST - 1 slabs fly while one is
// multiplied, one barrier per slab.  The window rows of a slab reach LDS the
// same way, into a ring of NST slots, issued with the operand loads NST - 1
// slabs before the ones that read them (so that waiting for a slab's operands
// also covers the window rows of the slab NST - 1 after it).  Every wave issues
// the same number of window-row loads per slab (unused ones read zero into a
// spare row), which keeps the wait counts compile-time constants.
template <class C, int BKS, int NST>
__global__ void __launch_bounds__(C::NT) k_wgrad_tr(WGradGroup grp, ExtraTask x) {
  using T = __bf16;
  constexpr int BM = C::BM, BN = C::BN, NT = C::NT, BK = C::BK;
  static_assert(NT == 256 && BM == 128 && BK % BKS == 0 && BKS % C::KB == 0 && NST >= 2 && NST <= 4,
                "slab and thread layout below");
  constexpr int ACH = BM / 8, BCH = BN / 8;  // 16-byte chunks per LDS row
  constexpr int AV = BKS * ACH / NT, BV = BKS * BCH / NT;
  static_assert(AV * NT == BKS * ACH && BV * NT == BKS * BCH, "slab splits evenly over the threads");
  constexpr int LPS = AV + BV;                       // operand loads per thread and slab
  constexpr int STG = BKS * (BM + BN);               // elements per stage
  // window-row entries per slab, rounded up to whole 64-dword loads: a load's
  // lanes past the slab's entries still write (zeros) to LDS
  constexpr int RSLOT = (BKS * AMAX + 63) / 64 * 64;
  constexpr int NRW = (RSLOT / 64 + 3) / 4;          // window-row loads per wave and slab
  __shared__ __attribute__((aligned(16))) T smem[NST * STG];
  __shared__ __attribute__((aligned(16))) int32_t Rr[NST * RSLOT + 64];  // + a spare row for unused loads

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / C::WN, wn = wave % C::WN;
  if (run_extra<T>(x)) return;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t lds_s = lds_addr(smem), lds_r = lds_addr(Rr), lds_spare = lds_r + NST * RSLOT * 4;
  // this thread's 16-byte LDS slots, the same in every slab: A rows tid / ACH +
  // j NT / ACH at slot tid % ACH, B rows tid / BCH + j NT / BCH at slot tid % BCH
  // (the row bits the swizzle reads do not change with j), and the logical
  // column chunk each slot holds
  const int ra0 = tid / ACH, ta = tid % ACH, rb0 = tid / BCH, tb = tid % BCH;
  const int ca = 2 * ((ta >> 1) ^ site_row_swz<BM * 2>(ra0)) + (ta & 1);
  const int cb = 2 * ((tb >> 1) ^ site_row_swz<BN * 2>(rb0)) + (tb & 1);

  for (int t = blockIdx.x; t < grp.tile_beg[grp.n]; t += own_grid(x)) {
    int l = 0;
    while (l + 1 < grp.n && t >= grp.tile_beg[l + 1]) ++l;
    const WGradArgs& a = grp.L[l];
    const int tile = t - grp.tile_beg[l];
    const int rows = a.rows_dev ? (*a.rows_dev + a.rows_add) : a.rows_host;
    const int tiles_m = a.Mpad / BM, tiles_n = a.Npad / BN;
    const int nch = wgrad_chunks_dev(a, rows, BK);
    const int per = ((rows + nch - 1) / nch + BK - 1) / BK * BK;
    const int m_gather = a.A * a.cseg;
    const int m_rows = a.m_ones >= 0 ? a.m_ones + 1 : m_gather;  // rows of dW / db that are read back
    const int tn = tile % tiles_n;
    const int tq = tile / tiles_n;
    const int tm = tq % tiles_m;
    const int chunk = tq / tiles_m;
    if (chunk >= nch) continue;  // fewer rows than the plan allowed for
    const int m0 = tm * BM, n0 = tn * BN;
    const int o_beg = chunk * per;
    const int o_end = min(rows, o_beg + per);
    const int nsl = o_end > o_beg ? (o_end - o_beg + BKS - 1) / BKS : 0;
    f32x4 acc[C::TM][C::TN];
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
      for (int j = 0; j < C::TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int A = a.A;
    const int ma = m0 + 8 * ca;  // first column of this thread's A chunk: window position fa, channel cola
    const bool a_col = ma < m_gather;
    const int fa = a_col ? ma / a.cseg : 0;
    const int cola = ma - fa * a.cseg;
    const int nb = n0 + 8 * cb;
    const bool b_col = nb < a.dsrc_cols;
    const bool has_r = a.rmap != nullptr;
    const int r_loads = has_r ? (BKS * A + 63) / 64 : 0;  // 64-dword loads that carry window rows
    // (held in registers: the loop's compiler fences would otherwise reload
    // them from the kernel arguments on every slab)
    const int src_stride = a.src_stride, dsrc_stride = a.dsrc_stride;
    const u32x4 rsA = buffer_rsrc(a.src, GATHER_SRC_BYTES);
    const u32x4 rsB = buffer_rsrc(a.dsrc, GATHER_SRC_BYTES);
    const u32x4 rsR = buffer_rsrc(a.rmap, GATHER_SRC_BYTES);
    const float rcpA = 1.f / (float)A;
    // window rows of slab s (sites ob .. ob + BKS - 1, A entries each,
    // contiguous) into ring slot s % NST: wave w's i-th load takes dwords
    // 64 k .. 64 k + 63, k = w + 4 i; NRW loads per wave whatever A and s
    auto issue_rows = [&](int s) {
      const int ob = o_beg + s * BKS;
      const uint32_t dst = lds_r + (uint32_t)((s % NST) * RSLOT) * 4u;
#pragma unroll
      for (int i = 0; i < NRW; ++i) {
        const int k = wave_u + 4 * i;
        const bool used = s < nsl && k < r_loads;
        const int d = 64 * k + lane;
        const bool live = used && d < BKS * A && ob + div_small(d, A, rcpA) < o_end;
        dma4(rsR, used ? dst + (uint32_t)k * 256u : lds_spare, live ? (uint32_t)(ob * A + d) * 4u : GATHER_SRC_BYTES);
      }
    };
    // operand slab s into stage s % NST, reading its window rows from ring slot s % NST
    auto issue_slab = [&](int s) {
      const int ob = o_beg + s * BKS;
      const uint32_t sa = lds_s + (uint32_t)((s % NST) * STG) * 2u, sb = sa + BM * BKS * 2;
      const int32_t* R = Rr + (s % NST) * RSLOT;
      uint32_t offa[AV];
#pragma unroll
      for (int j = 0; j < AV; ++j) {  // every window row read before the first load goes out
        const int r = ra0 + j * (NT / ACH);
        const int o = ob + r;
        const int srow = has_r ? R[r * A + fa] : o;
        offa[j] = a_col && o < o_end ? (uint32_t)(srow * src_stride + cola) * 2u : GATHER_SRC_BYTES;
      }
#pragma unroll
      for (int j = 0; j < AV; ++j) dma16(rsA, sa + (uint32_t)(wave_u * 64 + j * NT) * 16u, offa[j]);
#pragma unroll
      for (int j = 0; j < BV; ++j) {
        const int o = ob + rb0 + j * (NT / BCH);
        dma16(rsB, sb + (uint32_t)(wave_u * 64 + j * NT) * 16u,
              b_col && o < o_end ? (uint32_t)(o * dsrc_stride + nb) * 2u : GATHER_SRC_BYTES);
      }
    };
    // the bias row (softmax layer): the wave whose rows hold it patches its operand
    const int m_loc = a.m_ones - m0;
    const bool ones = a.m_ones >= 0 && m_loc >= wm * C::TM * 16 && m_loc < (wm + 1) * C::TM * 16;

    if (nsl > 0) {
      // window rows of the first NST - 1 slabs, their operands, then (once
      // every wave has read those ring slots) the window rows of the next NST - 1
      for (int p = 0; p < NST - 1; ++p) issue_rows(p);
      asm volatile("" ::: "memory");
      wait_vmcnt<0>();
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
      for (int p = 0; p < NST - 1; ++p)
        if (p < nsl) issue_slab(p);
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0) only: the operand loads stay in flight
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
      for (int p = NST - 1; p < 2 * NST - 2; ++p) issue_rows(p);
    }
    // the slab loop, with the bias-row patch compiled into a copy of its own
    // (a branch per slab made the compiler copy the accumulators between the
    // two MFMA sequences on every slab)
    auto slab_loop = [&](auto ones_c) {
      constexpr bool ONES = decltype(ones_c)::value;
      for (int s = 0; s < nsl; ++s) {
        // slab s and the window rows of slab s + NST - 1 have landed (this
        // wave's, and after the barrier every wave's); every wave is done with
        // slab s - 1 and with the ring slot refilled below.  Loads issued after
        // those may stay in flight: the window rows issued since (NRW per slab)
        // and the operand slabs after s that exist.
        asm volatile("" ::: "memory");
        if constexpr (NST == 2) {
          wait_vmcnt<0>();
        } else {
          // issued after the last load slab s needs (its operands, or at s <=
          // NST - 2 the prologue's window rows of slab s + NST - 1): NST - 2
          // batches of window rows, and the operand slabs i + NST - 1 < nsl
          // issued by iterations i = max(0, s - NST + 2) .. s - 1
          const int lo = max(0, s - NST + 2), hi = min(s - 1, nsl - NST);
          wait_vmcnt_steps<(NST - 2) * NRW, LPS>(hi >= lo ? hi - lo + 1 : 0);
        }
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        issue_rows(s + 2 * NST - 2);
        if (s + NST - 1 < nsl) issue_slab(s + NST - 1);
        const T* As = smem + (s % NST) * STG;
        const int valid = o_end - (o_beg + s * BKS);
        mma_slab_tr<C, BKS, ONES>(As, As + BM * BKS, acc, wm, wn, lane, m_loc, valid);
      }
    };
    if (ones)
      slab_loop(std::integral_constant<bool, true>{});
    else
      slab_loop(std::integral_constant<bool, false>{});

    store_wgrad_tile<C>(a, acc, chunk, nch, m0, n0, wm, wn, lane, m_rows, m_gather);
  }
}

// dW (and db) from the split-K partials, for a group of layers (block b
// belongs to layer l with blk_beg[l] <= b < blk_beg[l + 1]).  A block has G
// thread groups (G = 16, or fewer when there are fewer chunks) of 256/G
// threads, one 16-byte fragment quad of the partial layout (rows 4 g .. 4 g + 3
// of one column) per thread of a group; group g sums chunks g, g+G, ...; the G
// group sums are added in a fixed order.
__global__ void __launch_bounds__(256) k_wgrad_reduce(WGradGroup grp) {
  __shared__ f32x4 red[256];
  int l = 0;
  while (l + 1 < grp.n && (int)blockIdx.x >= grp.blk_beg[l + 1]) ++l;
  const WGradArgs& a = grp.L[l];
  const int nch = wgrad_chunks_dev(a, a.rows_dev ? (*a.rows_dev + a.rows_add) : a.rows_host, grp.BK);
  if (nch <= 1) return;  // the weight-gradient kernel wrote the results
  const int G = grp.G[l];
  const int E = 256 / G;  // quads per block
  const int m_gather = a.A * a.cseg;
  const int m_rows = a.m_ones >= 0 ? a.m_ones + 1 : m_gather;
  const int MB = (m_rows + 15) / 16, NB = (a.c_out + 15) / 16;
  const int64_t total = (int64_t)MB * NB * 64;
  const int el = threadIdx.x % E, grpi = threadIdx.x / E;
  const int64_t t = (int64_t)((int)blockIdx.x - grp.blk_beg[l]) * E + el;
  f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
  if (t < total) {
    const float* part = a.part + t * 4;
    const int64_t cstride = total * 4;
    for (int ch = grpi; ch < nch; ch += G) s += *(const f32x4*)(part + ch * cstride);
  }
  red[threadIdx.x] = s;
  __syncthreads();
  if (grpi != 0 || t >= total) return;
  s = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int g = 0; g < G; ++g) s += red[g * E + el];
  const int blk = (int)(t >> 6), ln = (int)(t & 63);
  const int bm = blk / NB, bn = blk - bm * NB;
  const int n = 16 * bn + (ln & 15);
  if (n >= a.c_out) return;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int m = 16 * bm + 4 * (ln >> 4) + r;
    if (m < m_gather) {
      const int f = m / a.cseg, c = m - f * a.cseg;
      if (c < a.c_in) a.dW[((int64_t)f * a.c_in + c) * a.c_out + n] = s[r];
    } else if (m == a.m_ones) {
      if (a.db) a.db[n] = s[r];
    }
  }
}

template <typename T>
__global__ void __launch_bounds__(256) k_row0_dx(Row0Args r) {
  row0_dx_block<T>(r, blockIdx.x);
}

static int device_grid_limit() { return 256 * 8; }

template <typename T, class C>
static void launch_cfg(const GemmArgs& a, int64_t max_rows, hipStream_t st) {
  const int64_t span = max_rows - a.row_begin;
  const int64_t tiles = ((span + C::BM - 1) / C::BM) * (a.Npad / C::BN) * a.ksplit;
  const int grid = (int)std::min<int64_t>(std::max<int64_t>(tiles, 1), device_grid_limit()) +
                   (a.x.kind ? a.x.blocks : 0);
  const bool timed = a.t_start || a.t_stop;
  // the pooling-backward epilogue and the masked store have instantiations of
  // their own (their extra loads and sums would otherwise cost every launch
  // registers)
  void (*kern)(GemmArgs) = a.pool_fwd ? k_gemm_gather<T, C, POOL_FWD_MODE>
                           : a.epi == EPI_STORE_MASK ? k_gemm_gather<T, C, MASK_MODE>
                           : !a.route ? k_gemm_gather<T, C, -1>
                           : a.route_ac == 4 ? k_gemm_gather<T, C, 4>
                                             : k_gemm_gather<T, C, 0>;
  const size_t lds = (size_t)C::BM * a.A * sizeof(int32_t);  // the window table: a workgroup's LDS follows A
  if (timed)
    hipExtLaunchKernelGGL(kern, dim3(grid), dim3(C::NT), lds, st, a.t_start,
                          a.ksplit > 1 && !a.partials_only ? nullptr : a.t_stop, 0, a);
  else
    hipLaunchKernelGGL(kern, dim3(grid), dim3(C::NT), lds, st, a);
  if (a.ksplit > 1 && !a.partials_only) {
    const int64_t total = span * ((a.out_cols + 3) / 4);
    const int g2 = (int)std::min<int64_t>(std::max<int64_t>((total + 255) / 256, 1), 4096);
    if (timed)
      hipExtLaunchKernelGGL(k_gemm_splitk_reduce<T>, dim3(g2), dim3(256), 0, st, nullptr, a.t_stop, 0, a);
    else
      hipLaunchKernelGGL(k_gemm_splitk_reduce<T>, dim3(g2), dim3(256), 0, st, a);
  }
}

template <typename T>
static void launch_gemm_t(const GemmArgs& a, int64_t max_rows, hipStream_t st) {
  switch (a.cfg) {
    case 0: launch_cfg<T, C128x128<T>>(a, max_rows, st); break;
    case 1: launch_cfg<T, C128x64<T>>(a, max_rows, st); break;
    case 2: launch_cfg<T, C64x64<T>>(a, max_rows, st); break;
    default: launch_cfg<T, C32x64<T>>(a, max_rows, st); break;
  }
}

hipError_t launch_gemm(bool bf16, const GemmArgs& args, int64_t max_rows, hipStream_t st) {
  if (max_rows - args.row_begin <= 0) return hipSuccess;
  if (max_rows > INT32_MAX) return hipErrorInvalidValue;
  if (args.A < 1 || args.A > AMAX) return hipErrorInvalidValue;  // window tables hold at most AMAX entries a row
  GemmArgs a = args;
  a.rows_cap = (int32_t)max_rows;
  if (a.pool_fwd && (a.route || a.ksplit != 1 || !gemm_routes(bf16, a.cfg) || a.row_begin != 0 || !a.pslot ||
                     !a.pool_out || !a.pool_argmax || !a.rows_dev ||
                     (a.epi != EPI_BIAS_RELU && a.epi != EPI_BIAS_LRELU)))
    return hipErrorInvalidValue;
  if (a.route) {  // pooling backward in the epilogue: one partial per row tile
    const int bm = gemm_bm(bf16, a.cfg);
    if (a.epi != EPI_STORE || a.ksplit != 1 || !gemm_routes(bf16, a.cfg) || (a.route_ac != 0 && a.route_ac != 4) ||
        !a.pr.part || !a.pr.Rp || !a.pr.argmax || !a.pr.dZ || !a.pr.X_pool || (a.route_ac == 4 && !a.pr.gmask) ||
        a.pr.cp != a.out_cols || a.pr.stride != a.pr.cp || (max_rows - a.row_begin + bm - 1) / bm > a.pr.PM)
      return hipErrorInvalidValue;
  }
  if (a.cfg == GEMM_DIRECT) return bf16 ? launch_gemm_direct(a, max_rows, st) : hipErrorInvalidValue;
  if (bf16)
    launch_gemm_t<__bf16>(a, max_rows, st);
  else
    launch_gemm_t<float>(a, max_rows, st);
  return hipGetLastError();
}

GemmPlan plan_gemm(bool bf16, int64_t max_rows, int N, int K, bool short_rows, int direct_max) {
  // bf16 launches with few output tiles (at the row bound) go to the
  // direct-operand kernel, whose waves split K and so keep many loads in flight
  // per tile; launches with more tiles keep the LDS-tiled kernel, whose slabs
  // stream through LDS stages shared by the tile's waves.  (Measured on the
  // pen-stroke DeepCNet(5,50), bf16, batch 100, tiles counted as 32 x 64 at the
  // row bound: input gradients with the pooling backward, direct 18.7 us against
  // 19.6 us at 316 tiles, but 24.1 against 20.4 at 1.1k and 31.1 against 20.9
  // at 3.3k; forward with the pooling forward even at 204 tiles; the softmax
  // layer's forward, 236 tiles, 7.2 us direct against 6.6 LDS-tiled.  The
  // callers pass 600, 256 and 128.)
  const int64_t direct_tiles = ((max_rows + DIRECT_BM - 1) / DIRECT_BM) * ((N + DIRECT_BN - 1) / DIRECT_BN);
  if (bf16 && direct_tiles <= direct_max && K <= 2048) {
    // waves per tile so that each sums at most about four 32-wide k blocks,
    // and more while the grid stays small
    GemmPlan p;
    p.cfg = GEMM_DIRECT;
    p.BN = DIRECT_BN;
    p.Npad = (int)round_up(N, DIRECT_BN);
    p.Kpad = (int)round_up(K, 64);
    p.ksplit = 1;
    const int ksteps = (K + 31) / 32;
    const int64_t tiles = ((max_rows + DIRECT_BM - 1) / DIRECT_BM) * (p.Npad / DIRECT_BN);
    int sk = 1;
    while (sk < 4 && sk * 4 < ksteps) sk *= 2;
    while (sk < 4 && sk * 2 <= ksteps && tiles * sk < 4096) sk *= 2;
    p.sk = sk;
    return p;
  }
  // Tile width: 128 when that pads N no more than 64 does and still gives >= 256
  // tiles; otherwise 64-wide tiles with the tallest of 128/64/32 rows that gives
  // >= 256 tiles.  K is split when even 32-row tiles leave the GPU mostly idle.
  // short_rows (an epilogue that routes every row through its pooling window,
  // a thread's rows one after another): at most 64 rows per tile, so that each
  // thread routes two rows, not four or eight (measured on the pen-stroke
  // DeepCNet(5,50) input gradient of the second level: 31.9 -> 25.8 us).
  const int BK = bf16 ? 64 : 32;
  const int64_t n128 = (N + 127) / 128 * 128, n64 = (N + 63) / 64 * 64;
  auto tiles = [&](int bm, int64_t npad, int bn) { return ((max_rows + bm - 1) / bm) * (npad / bn); };
  GemmPlan p;
  if (!short_rows && n128 <= n64 && tiles(128, n128, 128) >= 256)
    p.cfg = 0;
  else if (!short_rows && tiles(128, n64, 64) >= 256)
    p.cfg = 1;
  else if (tiles(64, n64, 64) >= 256)
    p.cfg = 2;
  else
    p.cfg = 3;
  const GemmTile t = gemm_tile(bf16, p.cfg);
  p.BN = t.BN;
  p.Npad = (int)round_up(N, t.BN);
  p.Kpad = (int)round_up(K, BK);
  const int64_t tl = tiles(t.BM, p.Npad, t.BN);
  const int kslabs = p.Kpad / BK;
  p.ksplit = 1;
  if (tl < 128 && kslabs >= 4) p.ksplit = (int)std::max<int64_t>(1, std::min<int64_t>(kslabs / 2, (256 + tl - 1) / tl));
  return p;
}

// sites per slab and LDS stages of the bf16 weight-gradient tiles
#ifndef WG_SLAB_128
#define WG_SLAB_128 32
#define WG_STAGES_128 4
#define WG_SLAB_64 32
#define WG_STAGES_64 3
#endif

hipError_t launch_wgrad(bool bf16, int cfg, const WGradArgs* layers, int n, hipStream_t st, const ExtraTask* extra) {
  // cfg: 0 = 128 x 128 tiles, 1 = 128 x 64
  if (n < 1 || n > MAX_WG_LAYERS) return hipErrorInvalidValue;
  const ExtraTask x = extra ? *extra : ExtraTask{};
  if (x.kind && (x.blocks < 1 || (x.kind != 1 && x.kind != 3))) return hipErrorInvalidValue;
  const int BN = cfg == 0 ? 128 : 64;
  WGradGroup g{};
  g.n = n;
  g.tile_beg[0] = 0;
  for (int l = 0; l < n; ++l) {
    if (layers[l].A < 1 || layers[l].A > AMAX) return hipErrorInvalidValue;
    g.L[l] = layers[l];
    g.tile_beg[l + 1] = g.tile_beg[l] + (layers[l].Mpad / 128) * (layers[l].Npad / BN) * layers[l].nchunks;
  }
  const int grid = std::min(std::max(g.tile_beg[n], 1), device_grid_limit()) + (x.kind ? x.blocks : 0);
  if (bf16) {
    if (cfg == 0)
      hipLaunchKernelGGL((k_wgrad_tr<C128x128<__bf16>, WG_SLAB_128, WG_STAGES_128>), dim3(grid), dim3(256), 0, st, g, x);
    else
      hipLaunchKernelGGL((k_wgrad_tr<C128x64<__bf16>, WG_SLAB_64, WG_STAGES_64>), dim3(grid), dim3(256), 0, st, g, x);
  } else {
    if (cfg == 0)
      hipLaunchKernelGGL((k_wgrad<float, C128x128<float>>), dim3(grid), dim3(256), 0, st, g, x);
    else
      hipLaunchKernelGGL((k_wgrad<float, C128x64<float>>), dim3(grid), dim3(256), 0, st, g, x);
  }
  return hipGetLastError();
}

hipError_t launch_wgrad_reduce(bool bf16, const WGradArgs* layers, int n, hipStream_t st) {
  WGradGroup g{};
  g.BK = bf16 ? 64 : 32;
  g.blk_beg[0] = 0;
  for (int l = 0; l < n; ++l) {
    const WGradArgs& a = layers[l];
    if (a.nchunks <= 1) continue;  // the weight-gradient kernel wrote the results
    const int m_rows = a.m_ones >= 0 ? a.m_ones + 1 : a.A * a.cseg;
    // fragment quads of the partial layout: 16 x 16 blocks over the rows and
    // columns read back, 64 per block
    const int64_t total = (int64_t)((m_rows + 15) / 16) * ((a.c_out + 15) / 16) * 64;
    const int G = a.nchunks >= 16 ? 16 : (a.nchunks >= 8 ? 8 : (a.nchunks >= 4 ? 4 : 2));
    const int E = 256 / G;
    g.L[g.n] = a;
    g.G[g.n] = G;
    g.blk_beg[g.n + 1] = g.blk_beg[g.n] + (int)((total + E - 1) / E);
    ++g.n;
  }
  if (g.n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_wgrad_reduce, dim3(g.blk_beg[g.n]), dim3(256), 0, st, g);
  return hipGetLastError();
}

hipError_t launch_row0_dx(bool bf16, const void* W, const float* D0, int32_t A, int32_t c_in, int32_t c_out,
                          int32_t cp_in, void* grad_in, const void* Y_below, float slope, hipStream_t st) {
  const Row0Args r{W, D0, A, c_in, c_out, cp_in, grad_in, Y_below, slope};
  if (bf16)
    hipLaunchKernelGGL(k_row0_dx<__bf16>, dim3(cp_in), dim3(256), 0, st, r);
  else
    hipLaunchKernelGGL(k_row0_dx<float>, dim3(cp_in), dim3(256), 0, st, r);
  return hipGetLastError();
}

}  // namespace sscn
