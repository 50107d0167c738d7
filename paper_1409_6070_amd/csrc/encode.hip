// Input encoding of online pen strokes (Section 2.4): per grid square the
// picture of the pen's path plus an 8-bin histogram of its movement in the 8
// compass directions, M = 9 features per site, sparse because squares the pen
// never touches carry nothing.
//
// Raster: consecutive points p0, p1 of a stroke are joined by pixels
// p0 + round_half_up(i * d / L), i = 0 .. L, d = p1 - p0, L = max(|dy|, |dx|)
// (8-connected).  Every unit move between consecutive pixels is one of E, NE, N,
// NW, W, SW, S, SE (counter-clockwise, north = -y); its length (1 or sqrt 2) is
// shared equally by the two squares it joins.  Direction channels are kept as
// integer move counts (integer atomics: the result does not depend on the order
// in which moves land) and turned into features at the end.

#include "common.h"
#include "kernels.h"

namespace sscn {

constexpr int ENC_THREADS = 256;

// floor(a / b) for b > 0
__device__ inline int floor_div(int a, int b) {
  const int q = a / b;
  return (a % b != 0 && a < 0) ? q - 1 : q;
}

// pixel i of the segment p0 -> p0 + d with L steps
__device__ inline int raster_coord(int p0, int d, int i, int L) { return p0 + floor_div(2 * i * d + L, 2 * L); }

// direction index of a unit move (dy, dx), -1 for no move
__device__ inline int move_dir(int dy, int dx) {
  constexpr int table[9] = {3, 2, 1, 4, -1, 0, 5, 6, 7};  // (dy + 1) * 3 + (dx + 1)
  return table[(dy + 1) * 3 + (dx + 1)];
}

// Stroke of point t: the last s with begin[s] <= t (empty strokes are skipped
// because their successor has the same begin); always in [0, n_strokes).
__device__ inline int stroke_of(const int32_t* begin, int n_strokes, int t) {
  int lo = 0, hi = n_strokes - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (begin[mid] <= t)
      lo = mid;
    else
      hi = mid - 1;
  }
  return lo;
}

__device__ inline bool in_grid(int y, int x, int N) { return (unsigned)y < (unsigned)N && (unsigned)x < (unsigned)N; }

__global__ void __launch_bounds__(256) k_enc_clear(uint32_t* p, int64_t words) {
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < words; t += (int64_t)gridDim.x * blockDim.x)
    p[t] = 0u;
}

// Offsets and samples are valid: begin runs from 0 to n_points, non-decreasing;
// every stroke's sample lies in the batch.
__global__ void __launch_bounds__(256) k_enc_check(EncodeArgs a) {
  for (int s = blockIdx.x * blockDim.x + threadIdx.x; s <= a.n_strokes; s += gridDim.x * blockDim.x) {
    const int b0 = a.begin[s];
    bool ok = b0 >= 0 && b0 <= a.n_points;
    if (s == 0) ok = ok && b0 == 0;
    if (s == a.n_strokes) ok = ok && b0 == a.n_points;
    if (s < a.n_strokes) {
      ok = ok && a.begin[s + 1] >= b0;
      if ((unsigned)a.sample[s] >= (unsigned)a.batch) atomicOr(a.err, ERRBIT_RANGE);
    }
    if (!ok) atomicOr(a.err, ERRBIT_ORDER);
  }
}

// Segment t -> t + 1 of its stroke (or the lone last point), validated; returns
// false when there is nothing to raster.
struct Seg {
  int b, y0, x0, dy, dx, L;
};
__device__ inline bool load_segment(const EncodeArgs& a, int t, Seg& g) {
  const int s = stroke_of(a.begin, a.n_strokes, t);
  const int end = min(a.begin[s + 1], a.n_points);
  g.b = a.sample[s];
  if ((unsigned)g.b >= (unsigned)a.batch || t >= end) return false;
  g.y0 = a.points[2 * t];
  g.x0 = a.points[2 * t + 1];
  if (!in_grid(g.y0, g.x0, a.N)) {
    atomicOr(a.err, ERRBIT_RANGE);
    return false;
  }
  g.dy = g.dx = g.L = 0;
  if (t + 1 < end) {
    const int y1 = a.points[2 * t + 2], x1 = a.points[2 * t + 3];
    if (in_grid(y1, x1, a.N)) {  // else: reported by that point's own thread; p0 alone is marked
      g.dy = y1 - g.y0;
      g.dx = x1 - g.x0;
      g.L = max(abs(g.dy), abs(g.dx));
    }
  }
  return true;
}

// Marks pixels 0 .. L-1 of every segment and the last point of every stroke.
__global__ void __launch_bounds__(256) k_enc_mark(EncodeArgs a) {
  for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < a.n_points; t += gridDim.x * blockDim.x) {
    Seg g;
    if (!load_segment(a, t, g)) continue;
    const int last = g.L == 0 ? 0 : g.L - 1;
    for (int i = 0; i <= last; ++i) {
      const int y = g.L ? raster_coord(g.y0, g.dy, i, g.L) : g.y0;
      const int x = g.L ? raster_coord(g.x0, g.dx, i, g.L) : g.x0;
      const int64_t w = ((int64_t)g.b * a.N + y) * a.Wd + (x >> 6);
      atomicOr((unsigned long long*)&a.bits[w], 1ull << (x & 63));
    }
  }
}

// Per sample: exclusive popcount prefix of its words (wpre) and its site count.
__global__ void __launch_bounds__(ENC_THREADS) k_enc_prefix(EncodeArgs a) {
  __shared__ int scratch[ENC_THREADS];
  const int b = blockIdx.x, t = threadIdx.x;
  const int nw = a.N * a.Wd;
  const uint64_t* w = a.bits + (int64_t)b * nw;
  int32_t* pre = a.wpre + (int64_t)b * nw;
  const int per = (nw + ENC_THREADS - 1) / ENC_THREADS;
  const int beg = t * per;
  int local = 0;
  for (int j = 0; j < per; ++j)
    if (beg + j < nw) local += __popcll(w[beg + j]);
  scratch[t] = local;
  __syncthreads();
  for (int off = 1; off < ENC_THREADS; off <<= 1) {
    const int v = t >= off ? scratch[t - off] : 0;
    __syncthreads();
    scratch[t] += v;
    __syncthreads();
  }
  int run = scratch[t] - local;
  for (int j = 0; j < per; ++j)
    if (beg + j < nw) {
      pre[beg + j] = run;
      run += __popcll(w[beg + j]);
    }
  if (t == ENC_THREADS - 1) a.scount[b] = scratch[ENC_THREADS - 1];
}

// Sample offsets (exclusive scan of the counts) and the total, one workgroup.
__global__ void __launch_bounds__(ENC_THREADS) k_enc_offsets(EncodeArgs a) {
  __shared__ int scratch[ENC_THREADS];
  const int t = threadIdx.x;
  const int per = (a.batch + ENC_THREADS - 1) / ENC_THREADS;
  const int beg = t * per;
  int local = 0;
  for (int j = 0; j < per; ++j)
    if (beg + j < a.batch) local += a.scount[beg + j];
  scratch[t] = local;
  __syncthreads();
  for (int off = 1; off < ENC_THREADS; off <<= 1) {
    const int v = t >= off ? scratch[t - off] : 0;
    __syncthreads();
    scratch[t] += v;
    __syncthreads();
  }
  int run = scratch[t] - local;
  for (int j = 0; j < per; ++j)
    if (beg + j < a.batch) {
      a.soff[beg + j] = run;
      run += a.scount[beg + j];
    }
  if (t == ENC_THREADS - 1) a.total[0] = scratch[ENC_THREADS - 1];
}

// Row (0-based) of the marked pixel (b, y, x).
__device__ inline int enc_row(const EncodeArgs& a, int b, int y, int x) {
  const int64_t idx = ((int64_t)b * a.N + y) * a.Wd + (x >> 6);
  const uint64_t below = a.bits[idx] & ((1ull << (x & 63)) - 1ull);
  return a.soff[b] + a.wpre[idx] + __popcll(below);
}

// Sites in ascending (b, y, x) order, the first max_sites of them.
__global__ void __launch_bounds__(256) k_enc_sites(EncodeArgs a) {
  const int nw = a.N * a.Wd;
  const int64_t words = (int64_t)a.batch * nw;
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < words; g += (int64_t)gridDim.x * blockDim.x) {
    uint64_t w = a.bits[g];
    if (!w) continue;
    const int b = (int)(g / nw);
    const int rem = (int)(g - (int64_t)b * nw);
    const int y = rem / a.Wd, wx = rem - y * a.Wd;
    int row = a.soff[b] + a.wpre[g];
    while (w) {
      const int bit = __ffsll((long long)w) - 1;
      w &= w - 1;
      if (row < a.max_sites) {
        a.coords[3 * (int64_t)row] = b;
        a.coords[3 * (int64_t)row + 1] = y;
        a.coords[3 * (int64_t)row + 2] = wx * 64 + bit;
      }
      ++row;
    }
  }
}

// Move counts: each unit move adds 1 to its direction at both squares it joins.
__global__ void __launch_bounds__(256) k_enc_moves(EncodeArgs a) {
  for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < a.n_points; t += gridDim.x * blockDim.x) {
    Seg g;
    if (!load_segment(a, t, g) || g.L == 0) continue;
    int py = g.y0, px = g.x0;
    int pr = enc_row(a, g.b, py, px);
    for (int i = 1; i <= g.L; ++i) {
      const int y = raster_coord(g.y0, g.dy, i, g.L), x = raster_coord(g.x0, g.dx, i, g.L);
      const int r = enc_row(a, g.b, y, x);
      const int d = move_dir(y - py, x - px);
      if (pr < a.max_sites) atomicAdd(&a.counts[8 * (int64_t)pr + d], 1);
      if (r < a.max_sites) atomicAdd(&a.counts[8 * (int64_t)r + d], 1);
      py = y;
      px = x;
      pr = r;
    }
  }
}

// Features: picture channel 1, direction channel d = count * length_d / 2.
template <typename T>
__global__ void __launch_bounds__(256) k_enc_feats(EncodeArgs a, T* feats) {
  const int64_t n = min(a.total[0], a.max_sites);
  const int64_t items = n * 9;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < items; t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = t / 9;
    const int c = (int)(t - r * 9);
    float v = 1.f;
    if (c > 0) {
      const int d = c - 1;
      v = (float)a.counts[8 * r + d] * ((d & 1) ? 0.70710678118654752f : 0.5f);
    }
    feats[t] = Elem<T>::from_f32(v);
  }
}

static int enc_grid(int64_t items) { return (int)std::max<int64_t>(1, std::min<int64_t>((items + 255) / 256, 4096)); }

hipError_t launch_encode(bool bf16, const EncodeArgs& a, void* feats, hipStream_t st) {
  const int64_t words = (int64_t)a.batch * a.N * a.Wd;
  // bitmap words and move counts start at zero; so does the error word
  hipLaunchKernelGGL(k_enc_clear, dim3(enc_grid(2 * words)), dim3(256), 0, st, (uint32_t*)a.bits, 2 * words);
  hipLaunchKernelGGL(k_enc_clear, dim3(enc_grid((int64_t)a.max_sites * 8)), dim3(256), 0, st, (uint32_t*)a.counts,
                     (int64_t)a.max_sites * 8);
  hipLaunchKernelGGL(k_enc_clear, dim3(1), dim3(256), 0, st, (uint32_t*)a.err, (int64_t)1);
  hipLaunchKernelGGL(k_enc_check, dim3(enc_grid(a.n_strokes + 1)), dim3(256), 0, st, a);
  if (a.n_points > 0 && a.n_strokes > 0)
    hipLaunchKernelGGL(k_enc_mark, dim3(enc_grid(a.n_points)), dim3(256), 0, st, a);
  if (a.batch > 0) {
    hipLaunchKernelGGL(k_enc_prefix, dim3(a.batch), dim3(ENC_THREADS), 0, st, a);
    hipLaunchKernelGGL(k_enc_offsets, dim3(1), dim3(ENC_THREADS), 0, st, a);
    hipLaunchKernelGGL(k_enc_sites, dim3(enc_grid(words)), dim3(256), 0, st, a);
  } else {
    hipLaunchKernelGGL(k_enc_clear, dim3(1), dim3(256), 0, st, (uint32_t*)a.total, (int64_t)1);
  }
  if (a.n_points > 0 && a.n_strokes > 0 && a.batch > 0)
    hipLaunchKernelGGL(k_enc_moves, dim3(enc_grid(a.n_points)), dim3(256), 0, st, a);
  const int grid = enc_grid((int64_t)a.max_sites * 9);
  if (bf16)
    hipLaunchKernelGGL(k_enc_feats<__bf16>, dim3(grid), dim3(256), 0, st, a, (__bf16*)feats);
  else
    hipLaunchKernelGGL(k_enc_feats<float>, dim3(grid), dim3(256), 0, st, a, (float*)feats);
  return hipGetLastError();
}

}  // namespace sscn
