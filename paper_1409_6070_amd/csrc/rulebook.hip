// Active-site sets and window lists for every layer (the paper's pointer
// matrices, Section 2.3), built on the GPU.
//
// Each layer's pointer matrix is held as an occupancy bitmap with one bit per
// grid location, rows aligned to 64-bit words, plus the exclusive popcount
// prefix of every word within its sample.  The row of an active location is
// then 1 + (sites in earlier samples) + (prefix of its word) + (set bits below
// it in the word): an order-preserving perfect hash of (b, y, x) onto rows
// 1..n, giving ascending (b, y, x) order with no sort.  Duplicates are found
// from the previous value returned by the atomic OR that inserts a site.
//
// Active sets follow Section 2.3 and Figure 2: a convolution output is active
// when any location of its FxF window below is active, a pooling output when
// any of its 2x2 stride-2 window is.  Composed down to the input, the windows
// of layer s cover one contiguous square: output (Y, X) is active iff an input
// site lies in [a Y, a Y + r - 1]^2, where a convolution adds a (F - 1) to r and
// a pooling layer adds a to r and doubles a (r >= a throughout, so the union of
// the windows below is contiguous).  Every layer's bitmap therefore comes
// straight from the input bitmap, one wave per (sample, layer), with no chain
// through the layers: the rows of each square are ORed word-parallel, then
// each output bit tests its column range.  The rows, window lists and
// transposes of a layer then come from one pass over its bitmap words: a
// workgroup lists its words' sites in row order in LDS and its threads take
// them one after another.  The sample offsets (exclusive scan of the
// per-sample counts) are scanned by every workgroup of that kernel for batches
// of up to 1024 samples; above that a separate offsets launch computes them (a
// last-workgroup pattern in the bitmap kernel would need a device-scope release
// fence, which costs more here than the launch).
//
// Builds alternate between two input bitmaps (and error words): each build
// inserts into one that is all zero and clears the other for the next build,
// so no clearing launch precedes the insertion.

#include "common.h"
#include "kernels.h"

namespace sscn {

// Clears both input bitmaps and the error and counter words (when a workspace
// is bound; afterwards each build clears what the next one needs).
__global__ void __launch_bounds__(256) k_rb_clear(uint64_t* bits_a, uint64_t* bits_b, int64_t nwords, int32_t* err) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (; i < nwords; i += stride) {
    bits_a[i] = 0ull;
    bits_b[i] = 0ull;
  }
  if (blockIdx.x == 0 && threadIdx.x < 4) err[threadIdx.x] = 0;
}

__global__ void __launch_bounds__(256) k_rb_insert(const int32_t* __restrict__ coords, int32_t n, int32_t batch,
                                                   int32_t N, int32_t Wd, uint64_t* bits0, int32_t* err) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  int b = coords[3 * i], y = coords[3 * i + 1], x = coords[3 * i + 2];
  if (b < 0 || b >= batch || y < 0 || y >= N || x < 0 || x >= N) {
    atomicOr(err, ERRBIT_RANGE);
    return;
  }
  unsigned long long bit = 1ull << (x & 63);
  unsigned long long* w = (unsigned long long*)&bits0[((int64_t)b * N + y) * Wd + (x >> 6)];
  unsigned long long old = atomicOr(w, bit);
  if (old & bit) atomicOr(err, ERRBIT_DUP);
}

__device__ inline uint64_t row_mask_word(int w, int S) {
  int lo = w * 64;
  int nb = S - lo;
  if (nb >= 64) return ~0ull;
  if (nb <= 0) return 0ull;
  return (1ull << nb) - 1ull;
}

// Exclusive prefix of one value per lane over a wave; *total gets the sum.
__device__ inline int wave_exclusive_scan(int v, int* total) {
  const int lane = threadIdx.x & 63;
  int x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int u = __shfl_up(x, off, 64);
    if (lane >= off) x += u;
  }
  *total = __shfl(x, 63, 64);
  return x - v;
}

// Popcount prefix of nw words held in LDS by one wave (lane t takes the
// contiguous words [t * per, (t + 1) * per)): writes wpre[0..nw) and returns
// the total.
__device__ inline int wave_popcount_scan(const uint64_t* words, int nw, int32_t* wpre) {
  const int t = threadIdx.x;
  const int per = (nw + 63) / 64;
  const int beg = min(nw, t * per), end = min(nw, beg + per);
  int local = 0;
  for (int w = beg; w < end; ++w) local += __popcll(words[w]);
  int total;
  int run = wave_exclusive_scan(local, &total);
  for (int w = beg; w < end; ++w) {
    wpre[w] = run;
    run += __popcll(words[w]);
  }
  return total;
}

// q = k / d for 0 <= k < 2^20, 1 <= d < 2^16 (rcp = 1/d): float estimate,
// then exact correction (an integer division by a runtime value costs tens of
// instructions).
__device__ inline int div_rcp(int k, int d, float rcp) {
  int q = (int)((float)k * rcp);
  q += (q + 1) * d <= k ? 1 : 0;
  q -= q * d > k ? 1 : 0;
  return q;
}

// q = k / d for 0 <= k < 2^40, 1 <= d < 2^20: double estimate, then exact
// correction.
__device__ inline int div_rcp_d(int64_t k, int d) {
  int64_t q = (int64_t)((double)k * (1.0 / (double)d));
  q += (q + 1) * d <= k ? 1 : 0;
  q -= q * d > k ? 1 : 0;
  return (int)q;
}

// Sites beg .. end - 1 of sample b into the sample's LDS bitmap `in` ([S0][W0]
// words) by atomic ORs, sixteen sites per lane in flight; returns the error
// bits (a site of another sample or off the grid; with DUP a site set twice).
template <bool DUP>
__device__ inline int insert_sample(const int32_t* coords, int beg, int end, int b, int S0, int W0, uint64_t* in) {
  constexpr int SPL = 16;
  int err = 0;
  for (int i0 = beg + (int)threadIdx.x; i0 < end; i0 += SPL * 64) {
    int cb[SPL], cy[SPL], cx[SPL];
#pragma unroll
    for (int u = 0; u < SPL; ++u) {
      const int64_t i = i0 + 64 * u < end ? i0 + 64 * u : beg;
      cb[u] = coords[3 * i];
      cy[u] = coords[3 * i + 1];
      cx[u] = coords[3 * i + 2];
    }
#pragma unroll
    for (int u = 0; u < SPL; ++u) {
      if (i0 + 64 * u >= end) break;
      if (cb[u] != b || cy[u] < 0 || cy[u] >= S0 || cx[u] < 0 || cx[u] >= S0) {
        err |= ERRBIT_RANGE;
        continue;
      }
      const unsigned long long bit = 1ull << (cx[u] & 63);
      unsigned long long* w = (unsigned long long*)&in[cy[u] * W0 + (cx[u] >> 6)];
      if constexpr (DUP) {
        if (atomicOr(w, bit) & bit) err |= ERRBIT_DUP;
      } else {
        __hip_atomic_fetch_or(w, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      }
    }
  }
  return err;
}

// Layer s of sample b, b = blockIdx / nlayers, s = blockIdx % nlayers (one
// wave): the sample's input bitmap goes to LDS (read from the inserted bitmap,
// or, with the sites grouped by sample, built here from the sample's own
// sites by LDS atomic ORs, the input layer's wave storing it); each lane takes whole output
// rows, ORs the input rows of their squares into its own row buffer, and sets
// each output bit whose column range of that row holds a set bit (a word-
// parallel dilation when a = 1).  Then the layer's word prefix and count, as
// the layer-by-layer definition gives them.  Every workgroup also clears its
// share of the next build's input bitmap; workgroups of samples b >= batch only
// clear.
__global__ void __launch_bounds__(64) k_rb_bitmaps(RulebookArgs a, int32_t max_words) {
  extern __shared__ uint64_t lds[];
  const LayerBits& L0 = a.L[0];
  const int S0 = L0.S, W0 = L0.Wd, nw0 = S0 * W0;
  uint64_t* in = lds;                      // [S0][W0]
  uint64_t* out = lds + max_words;         // [So][Wo]
  uint64_t* rowbuf = lds + 2 * max_words;  // [64][W0]
  const int s = (int)blockIdx.x % a.nlayers, b = (int)blockIdx.x / a.nlayers;
  const int t = threadIdx.x;
  {
    const int64_t total = (int64_t)a.batch_max * nw0;
    for (int64_t i = (int64_t)blockIdx.x * 64 + t; i < total; i += (int64_t)gridDim.x * 64) a.bits0_next[i] = 0ull;
    if (blockIdx.x == 0 && t == 0) *a.err_next = 0;
  }
  if (b >= a.batch) return;
  if (a.sample_begin) {
    // sites grouped by sample: this wave inserts sample b's sites into its own
    // LDS bitmap (every wave of the sample does; the input layer's reports
    // the errors and stores the bitmap for the window lists)
    for (int w = t; w < nw0; w += 64) in[w] = 0ull;
    __syncthreads();
    const int n = a.n;
    int beg = a.sample_begin[b], end = a.sample_begin[b + 1];
    const bool bad = beg < 0 || end < beg || end > n || (b == 0 && beg != 0) || (b == a.batch - 1 && end != n);
    beg = min(max(beg, 0), n);
    end = min(max(end, beg), n);
    int err;
    // the input layer's wave looks for duplicates in the values its ORs return;
    // the others need no returned value
    if (s == 0)
      err = insert_sample<true>(a.coords, beg, end, b, S0, W0, in);
    else
      err = insert_sample<false>(a.coords, beg, end, b, S0, W0, in);
    if (s == 0 && (err || (bad && t == 0))) atomicOr(a.err, err | (bad ? ERRBIT_RANGE : 0));
    __syncthreads();
    if (s == 0) {
      uint64_t* dst = L0.bits + (int64_t)b * nw0;
      for (int w = t; w < nw0; w += 64) dst[w] = in[w];
    }
  } else {
    const uint64_t* src = L0.bits + (int64_t)b * nw0;
    for (int w0 = t; w0 < nw0; w0 += 4 * 64) {  // four words per lane in flight
      uint64_t v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = src[min(w0 + u * 64, nw0 - 1)];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (w0 + u * 64 < nw0) in[w0 + u * 64] = v[u];
    }
    __syncthreads();
  }
  if (s == 0) {  // the input layer: its prefix and count only
    const int tot = wave_popcount_scan(in, nw0, L0.wpre + (int64_t)b * nw0);
    if (t == 0) L0.scount[b] = tot;
    return;
  }
  const LayerBits& Lo = a.L[s];
  const int Wo = Lo.Wd, So = Lo.S, nwo = So * Wo;
  const int ra = a.rf_a[s], rr = a.rf_r[s];
  uint64_t* row = rowbuf + t * W0;
  // P lanes per output row (a power of two, P * So <= 64 when So < 64): the
  // deep layers have few rows, each the OR of many input rows, which the P
  // lanes split and combine by shuffles
  const int P = So >= 64 ? 1 : 1 << (31 - __clz(64 / So));
  for (int Y0 = 0; Y0 < So; Y0 += 64 / P) {  // uniform over the wave
    const int Y = Y0 + t / P, sub = t % P;
    const bool live = Y < So;
    const int y_end = live ? min(ra * Y + rr, S0) : 0;
    for (int w = 0; w < W0; ++w) {  // OR of the square's input rows
      uint64_t v = 0;
#pragma unroll 4
      for (int y = ra * Y + sub; y < y_end; y += P) v |= in[y * W0 + w];
      for (int m = 1; m < P; m <<= 1) {
        const uint32_t lo = __shfl_xor((uint32_t)v, m, 64), hi = __shfl_xor((uint32_t)(v >> 32), m, 64);
        v |= ((uint64_t)hi << 32) | lo;
      }
      row[w] = v;
    }
    if (!live || sub) continue;
    if (ra == 1) {  // output bit X covers input bits X .. X + rr - 1
      for (int w = 0; w < Wo; ++w) {
        const uint64_t lo = row[w], hi = w + 1 < W0 ? row[w + 1] : 0ull;
        uint64_t acc = lo;
        for (int d = 1; d < rr; ++d) acc |= (lo >> d) | (hi << (64 - d));
        out[Y * Wo + w] = acc & row_mask_word(w, So);
      }
    } else if (W0 <= 2 && rr <= 64) {  // the input row in registers: bit X = any of bits [a X, a X + rr)
      const uint64_t r0 = row[0], r1 = W0 > 1 ? row[1] : 0ull;
      const uint64_t lmask = rr == 64 ? ~0ull : (1ull << rr) - 1ull;
      for (int w = 0; w < Wo; ++w) {
        uint64_t acc = 0;
        const int x_end = min(So, (w + 1) * 64);
#pragma unroll 4
        for (int x = w * 64; x < x_end; ++x) {
          const int lo = ra * x;  // < S0 <= 128; bits past S0 are zero
          const uint64_t v = lo < 64 ? (r0 >> lo) | (lo ? r1 << (64 - lo) : 0ull) : r1 >> (lo - 64);
          acc |= ((v & lmask) ? 1ull : 0ull) << (x - w * 64);
        }
        out[Y * Wo + w] = acc;
      }
    } else {  // output bit X covers input bits [a X, a X + rr)
      for (int w = 0; w < Wo; ++w) {
        uint64_t acc = 0;
        const int x_end = min(So, (w + 1) * 64);
#pragma unroll 4
        for (int x = w * 64; x < x_end; ++x) {
          const int lo = ra * x, hi = min(lo + rr, S0);
          const int wl = lo >> 6, wh = (hi - 1) >> 6;
          uint64_t any = 0;
          for (int q = wl; q <= wh; ++q) {
            uint64_t v = row[q];
            if (q == wl) v &= ~0ull << (lo & 63);
            if (q == wh && (hi & 63)) v &= (1ull << (hi & 63)) - 1ull;
            any |= v;
          }
          acc |= (any ? 1ull : 0ull) << (x - w * 64);
        }
        out[Y * Wo + w] = acc;
      }
    }
  }
  __syncthreads();
  uint64_t* dst = Lo.bits + (int64_t)b * nwo;
  for (int w = t; w < nwo; w += 64) dst[w] = out[w];
  const int tot = wave_popcount_scan(out, nwo, Lo.wpre + (int64_t)b * nwo);
  if (t == 0) Lo.scount[b] = tot;
}

// Sample offsets and layer totals: one wave per layer, an exclusive scan of the
// per-sample counts.
__global__ void __launch_bounds__(64) k_rb_offsets(RulebookArgs a) {
  const int s = blockIdx.x, t = threadIdx.x;
  const LayerBits& L = a.L[s];
  const int per = (a.batch + 63) / 64;
  const int beg = min(a.batch, t * per), end = min(a.batch, beg + per);
  int local = 0;
#pragma unroll 4
  for (int i = beg; i < end; ++i) local += L.scount[i];
  int total;
  int run = wave_exclusive_scan(local, &total);
  for (int i = beg; i < end; ++i) {
    L.soff[i] = run;
    run += L.scount[i];
  }
  if (t == 0) a.counts[s] = total;
}

// Batches up to this size have their sample offsets scanned inside the
// window-list kernel (no separate offsets launch).
constexpr int LISTS_SCAN_MAX = 1024;

// Exclusive prefixes of up to three count arrays sc[k][0, batch) (null: not
// scanned) into the LDS arrays off + k * batch, by one workgroup of 256
// threads (batch <= LISTS_SCAN_MAX): every count is loaded before the first
// is used.  Returns the total of sc[1] (or of sc[0] when nk == 1).  All threads
// call it; it synchronises before returning.
__device__ inline int block_count_scan(const int32_t* const (&sc)[3], int nk, int batch, int* off, int (*wsum)[4]) {
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int per = (batch + 255) / 256;  // <= 4
  const int beg = min(batch, t * per), end = min(batch, beg + per);
  int c[3][4];
#pragma unroll
  for (int k = 0; k < 3; ++k)
#pragma unroll
    for (int u = 0; u < 4; ++u) c[k][u] = k < nk && sc[k] && beg + u < end ? sc[k][beg + u] : 0;
  int run[3];
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    const int local = (c[k][0] + c[k][1]) + (c[k][2] + c[k][3]);
    int wt;
    run[k] = wave_exclusive_scan(local, &wt);
    if (lane == 0) wsum[k][wv] = wt;
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    if (k >= nk || !sc[k]) continue;
    for (int q = 0; q < wv; ++q) run[k] += wsum[k][q];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (beg + u < end) {
        off[k * batch + beg + u] = run[k];
        run[k] += c[k][u];
      }
  }
  const int kt = nk == 1 ? 0 : 1;
  const int total = (wsum[kt][0] + wsum[kt][1]) + (wsum[kt][2] + wsum[kt][3]);
  __syncthreads();
  return total;
}

// Row of location (y, x) of sample b in layer L (0 when inactive); off: the
// sample's offset (sites in earlier samples).
__device__ inline int32_t rank_row(const LayerBits& L, int b, int y, int x, int32_t off) {
  int64_t idx = ((int64_t)b * L.S + y) * L.Wd + (x >> 6);
  uint64_t w = L.bits[idx];
  int bit = x & 63;
  if (!((w >> bit) & 1ull)) return 0;
  return 1 + off + L.wpre[idx] + __popcll(w & ((1ull << bit) - 1ull));
}

// Rows of the F x F locations (y0 + SIGN*dy, x0 + SIGN*dx), dy, dx < F, of
// layer L in sample b (offset off): 0 where a location is inactive, `outside`
// where it lies off the grid.  Every word and prefix load is issued before any
// is used.
template <int F, int SIGN>
__device__ inline void rank_window(const LayerBits& L, int b, int y0, int x0, int32_t outside, int32_t off,
                                   int32_t (&r)[F * F]) {
  constexpr int A = F * F;
  int64_t idx[A];
  int bit[A];
  bool in[A];
#pragma unroll
  for (int dy = 0; dy < F; ++dy)
#pragma unroll
    for (int dx = 0; dx < F; ++dx) {
      const int f = dy * F + dx, y = y0 + SIGN * dy, x = x0 + SIGN * dx;
      in[f] = y >= 0 && x >= 0 && y < L.S && x < L.S;
      idx[f] = in[f] ? ((int64_t)b * L.S + y) * L.Wd + (x >> 6) : 0;
      bit[f] = x & 63;
    }
  uint64_t w[A];
  int32_t pre[A];
#pragma unroll
  for (int f = 0; f < A; ++f) {
    w[f] = L.bits[idx[f]];
    pre[f] = L.wpre[idx[f]];
  }
#pragma unroll
  for (int f = 0; f < A; ++f) {
    const bool on = (w[f] >> bit[f]) & 1ull;
    r[f] = !in[f] ? outside : on ? 1 + off + pre[f] + __popcll(w[f] & ((1ull << bit[f]) - 1ull)) : 0;
  }
}

// Child ground mask of pooling location (Y, X) of sample b over a 2x2
// convolution whose input is layer L: bit 4 f + k, for pooling position
// f = 2 dy + dx and convolution window position k = 2 ky + kx, is set when
// location (2Y + dy + ky, 2X + dx + kx) of L is inactive or off its grid, i.e.
// when that child's window reads the ground row there.  The nine locations
// are one 3x3 square: three rows of at most two words each.
__device__ inline uint16_t child_ground_mask(const LayerBits& L, int b, int Y, int X) {
  const int y0 = 2 * Y, x0 = 2 * X;
  const int wi = x0 >> 6, bi = x0 & 63;
  const bool two = bi > 61 && wi + 1 < L.Wd;
  uint64_t w0[3], w1[3];
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    const bool in = y0 + i < L.S && wi < L.Wd;
    const int64_t idx = ((int64_t)b * L.S + (in ? y0 + i : 0)) * L.Wd + (in ? wi : 0);
    w0[i] = in ? L.bits[idx] : 0ull;
    w1[i] = in && two ? L.bits[idx + 1] : 0ull;
  }
  uint32_t cols = 0;  // columns x0 .. x0 + 2 on the grid
#pragma unroll
  for (int j = 0; j < 3; ++j) cols |= (x0 + j < L.S ? 1u : 0u) << j;
  uint32_t act = 0;  // bit 3 i + j: location (y0 + i, x0 + j) active
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    const uint64_t v = (w0[i] >> bi) | (bi > 61 ? w1[i] << (64 - bi) : 0ull);
    act |= ((uint32_t)v & cols) << (3 * i);
  }
  uint32_t m = 0;
#pragma unroll
  for (int dy = 0; dy < 2; ++dy)
#pragma unroll
    for (int dx = 0; dx < 2; ++dx)
#pragma unroll
      for (int ky = 0; ky < 2; ++ky)
#pragma unroll
        for (int kx = 0; kx < 2; ++kx)
          m |= (((act >> (3 * (dy + ky) + dx + kx)) & 1u) ^ 1u) << (4 * (2 * dy + dx) + 2 * ky + kx);
  return (uint16_t)m;
}

// R_s of one row: the rows of layer Li under the F x F window of location
// (y, x) of sample b (locations step * (y, x) + (dy, dx)), 0 where inactive.
template <int F>
__device__ inline void row_window(const LayerBits& Li, int b, int y, int x, int step, int32_t off, int32_t* R) {
  int32_t r[F * F];
  rank_window<F, 1>(Li, b, step * y, step * x, 0, off, r);
#pragma unroll
  for (int f = 0; f < F * F; ++f) R[f] = r[f];
}

// Rt_s of one row of layer s - 1 at (y, x): the rows of layer Lo (a
// convolution) whose window holds it at each position, -1 where none.
template <int F>
__device__ inline void row_window_t(const LayerBits& Lo, int b, int y, int x, int32_t off, int32_t* Rt) {
  int32_t r[F * F];
  rank_window<F, -1>(Lo, b, y, x, -1, off, r);
#pragma unroll
  for (int f = 0; f < F * F; ++f) Rt[f] = r[f];
}

// Rows of every layer, their window lists and transposes, the caller-site ->
// row map and the head rows, in one launch.  Segment kind 0 (one per layer
// r): each workgroup takes LISTS_WPB consecutive bitmap words of layer r,
// eight threads per word, one byte each; the words' sites are listed in LDS
// in row order (row = 1 + sample offset + word prefix + rank in the word, a
// block scan over the threads' bytes), then every thread takes listed sites one after
// another and writes, for its site, the key (sites), R_r and the child ground
// mask (r >= 1), and the row's entries of Rt_{r+1} (r + 1 < nlayers).  Kind 2:
// caller site -> input row; kind 3: each sample's top-layer row.  SCAN: every
// workgroup scans the per-sample counts of the layers it looks up (dynamic
// LDS: three arrays of batch ints); otherwise the offsets kernel has stored
// them (soff) and the layer totals.

template <bool SCAN>
__global__ void __launch_bounds__(256) k_rb_lists(RulebookArgs a, ListsWork lw) {
  static_assert(LISTS_WPB * 8 == 256, "eight threads per bitmap word");
  extern __shared__ int32_t offs[];  // SCAN: [3][batch], layers r - 1, r, r + 1
  __shared__ int2 ent[LISTS_WPB * 64];
  __shared__ int wloc[LISTS_WPB][3];
  __shared__ int wsum[3][4];
  __shared__ int ntot;
  int seg = 0;
  while (seg + 1 < lw.nseg && (int)blockIdx.x >= lw.blk[seg + 1]) ++seg;
  const int kind = lw.kind[seg], r = lw.layer[seg];
  const int t = threadIdx.x;
  const int bi = (int)blockIdx.x - lw.blk[seg];
  const int B = a.batch;
  if (kind == 0) {
    const LayerBits& Lr = a.L[r];
    const bool lo = r >= 1, hi = r + 1 < a.nlayers;
    const int per_s = Lr.S * Lr.Wd;  // words per sample (< 2^20)
    const int64_t nwords = (int64_t)B * per_s;
    const int64_t w0 = (int64_t)bi * LISTS_WPB;
    // the words and prefixes do not depend on the offsets: loaded first.
    // Thread t takes bits 8 (t % 8) .. + 7 of word t / 8.
    const int wi = t >> 3, part = t & 7;
    uint64_t word = 0ull;
    int wp = 0;
    if (w0 + wi < nwords) {
      word = Lr.bits[w0 + wi];
      wp = Lr.wpre[w0 + wi];
    }
    int tot_r = 0;
    if constexpr (SCAN) {
      const int32_t* const sc[3] = {lo ? a.L[r - 1].scount : nullptr, Lr.scount, hi ? a.L[r + 1].scount : nullptr};
      tot_r = block_count_scan(sc, 3, B, offs, wsum);
    }
    auto off_of = [&](int which, int b) -> int32_t {  // which: 0 layer r - 1, 1 layer r, 2 layer r + 1
      if constexpr (SCAN)
        return offs[which * B + b];
      else
        return a.L[r - 1 + which].soff[b];
    };
    // list this workgroup's sites in row order: thread t's bits follow those
    // of threads < t (a block scan of the per-thread counts)
    const uint32_t mine = (uint32_t)(word >> (8 * part)) & 0xffu;
    int tw;
    int pre = wave_exclusive_scan(__popc(mine), &tw);
    if ((t & 63) == 0) wsum[0][t >> 6] = tw;
    __syncthreads();
    for (int q = 0; q < (t >> 6); ++q) pre += wsum[0][q];
    if (t == 0) ntot = (wsum[0][0] + wsum[0][1]) + (wsum[0][2] + wsum[0][3]);
    if (word) {
      const int64_t g = w0 + wi;
      const int b = div_rcp_d(g, per_s);
      if (part == 0) {
        const int rem = (int)(g - (int64_t)b * per_s);
        const int y = div_rcp(rem, Lr.Wd, 1.f / (float)Lr.Wd);
        wloc[wi][0] = b;
        wloc[wi][1] = y;
        wloc[wi][2] = (rem - y * Lr.Wd) * 64;
      }
      int row = 1 + off_of(1, b) + wp + __popcll(word & ((1ull << (8 * part)) - 1ull));
      int k = pre;
      uint32_t m = mine;
      while (m) {
        const int bit = __ffs(m) - 1;
        m &= m - 1;
        ent[k++] = make_int2(row++, wi * 64 + 8 * part + bit);
      }
    }
    __syncthreads();
    const int total = ntot;
    for (int i = t; i < total; i += blockDim.x) {
      const int2 e = ent[i];
      const int row = e.x, wt = e.y >> 6;
      const int b = wloc[wt][0], y = wloc[wt][1], x = wloc[wt][2] + (e.y & 63);
      Lr.sites[row - 1] = (b * Lr.S + y) * Lr.S + x;
      if (lo) {
        const LayerBits& Li = a.L[r - 1];
        const int F = a.F[r], step = a.kind[r] == 1 ? 1 : 2;
        const int32_t off = off_of(0, b);
        int32_t* R = a.rules[r] + (int64_t)row * F * F;
        if (F == 3)
          row_window<3>(Li, b, y, x, step, off, R);
        else if (F == 2)
          row_window<2>(Li, b, y, x, step, off, R);
        else
          row_window<1>(Li, b, y, x, step, off, R);
        if (r >= 2 && a.gmask[r]) a.gmask[r][row] = child_ground_mask(a.L[r - 2], b, y, x);
      }
      if (hi) {
        const LayerBits& Lo = a.L[r + 1];
        const int32_t off = off_of(2, b);
        if (a.kind[r + 1] == 1) {
          const int F = a.F[r + 1];
          int32_t* Rt = a.rules_t[r + 1] + (int64_t)row * F * F;
          if (F == 3)
            row_window_t<3>(Lo, b, y, x, off, Rt);
          else if (F == 2)
            row_window_t<2>(Lo, b, y, x, off, Rt);
          else
            row_window_t<1>(Lo, b, y, x, off, Rt);
        } else {  // pooling above: the parent's row times 4 plus the position in its window
          const int Y = y >> 1, X = x >> 1;
          int32_t p = -1;
          if (Y < Lo.S && X < Lo.S) p = rank_row(Lo, b, Y, X, off) * 4 + (y & 1) * 2 + (x & 1);
          a.rules_t[r + 1][row] = p;
        }
      }
    }
    if (bi == 0) {  // row 0 (the ground row) of every list this segment writes, and the layer's total
      if (lo) {
        const int A = a.F[r] * a.F[r];
        if (t < A) a.rules[r][t] = 0;
        if (t == 0 && r >= 2 && a.gmask[r]) a.gmask[r][0] = 0xFFFF;
      }
      if (hi) {
        const int At = a.kind[r + 1] == 1 ? a.F[r + 1] * a.F[r + 1] : 1;
        if (t < At) a.rules_t[r + 1][t] = -1;
      }
      if (SCAN && t == 0) a.counts[r] = tot_r;
    }
  } else if (kind == 2) {  // caller site -> input row
    const LayerBits& L0 = a.L[0];
    const int64_t i = (int64_t)bi * blockDim.x + t;
    int b = -1, y = 0, x = 0;
    if (i < a.n) {
      b = a.coords[3 * i];
      y = a.coords[3 * i + 1];
      x = a.coords[3 * i + 2];
    }
    if constexpr (SCAN) {
      const int32_t* const sc[3] = {L0.scount, nullptr, nullptr};
      block_count_scan(sc, 1, B, offs, wsum);
    }
    if (i < a.n) {
      int32_t p = -1;
      if (b >= 0 && b < B && y >= 0 && y < L0.S && x >= 0 && x < L0.S)
        p = rank_row(L0, b, y, x, SCAN ? offs[b] : L0.soff[b]);
      a.perm[i] = p;
    }
  } else {  // each sample's single top-layer site (row 0 when the sample is empty)
    const LayerBits& Lt = a.L[a.nlayers - 1];
    if constexpr (SCAN) {
      const int32_t* const sc[3] = {Lt.scount, nullptr, nullptr};
      block_count_scan(sc, 1, B, offs, wsum);
    }
    const int64_t b = (int64_t)bi * blockDim.x + t;
    if (b < B) a.head_rows[b] = rank_row(Lt, (int)b, 0, 0, SCAN ? offs[b] : Lt.soff[b]);
  }
}

hipError_t launch_rulebook(const RulebookArgs& a, const ListsWork& lw, int32_t max_words, hipStream_t st) {
  const LayerBits& L0 = a.L[0];
  if (a.n > 0 && !a.sample_begin)  // grouped sites: the bitmap kernel inserts them
    hipLaunchKernelGGL(k_rb_insert, dim3((a.n + 255) / 256), dim3(256), 0, st, a.coords, a.n, a.batch, L0.S, L0.Wd,
                       L0.bits, a.err);
  const size_t lds = (size_t)(2 * max_words + 64 * L0.Wd) * sizeof(uint64_t);
  hipLaunchKernelGGL(k_rb_bitmaps, dim3(std::max(a.batch, 1) * a.nlayers), dim3(64), lds, st, a, max_words);
  const bool scan = a.batch >= 1 && a.batch <= LISTS_SCAN_MAX;
  if (scan) {
    hipLaunchKernelGGL(k_rb_lists<true>, dim3(lw.blk[lw.nseg]), dim3(256), (size_t)3 * a.batch * sizeof(int32_t), st, a,
                       lw);
  } else {
    hipLaunchKernelGGL(k_rb_offsets, dim3(a.nlayers), dim3(64), 0, st, a);
    hipLaunchKernelGGL(k_rb_lists<false>, dim3(lw.blk[lw.nseg]), dim3(256), 0, st, a, lw);
  }
  return hipGetLastError();
}

hipError_t launch_rulebook_reset(uint64_t* bits_a, uint64_t* bits_b, int64_t nwords, int32_t* err, hipStream_t st) {
  const int g = (int)std::max<int64_t>(1, std::min<int64_t>((nwords + 255) / 256, 1024));
  hipLaunchKernelGGL(k_rb_clear, dim3(g), dim3(256), 0, st, bits_a, bits_b, nwords, err);
  return hipGetLastError();
}

}  // namespace sscn
