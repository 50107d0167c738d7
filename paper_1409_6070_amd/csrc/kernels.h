// Host-side launchers of the HIP kernels (internal to libsscn).
#pragma once

#include <algorithm>

#include "common.h"

namespace sscn {

// Bitmap words of a layer per workgroup of the window-list kernel.
constexpr int LISTS_WPB = 32;

// Segments of the window-list kernel: kind 0 = the rows of layer `layer`
// (their keys, R of that layer, the transposes of the layer above), with
// ceil(batch * S * Wd / LISTS_WPB) workgroups; 2 = caller-site rows and 3 = head
// rows, 256 per workgroup; segment i owns workgroups [blk[i], blk[i+1]).
struct ListsWork {
  int32_t nseg;
  int32_t kind[MAX_LAYERS + 2];
  int32_t layer[MAX_LAYERS + 2];
  int32_t blk[MAX_LAYERS + 3];
};

// Insertion, every layer's bitmap, then the window lists (with the sample
// offsets scanned in each workgroup for 1 <= batch <= 1024, else an offsets
// launch first).
hipError_t launch_rulebook(const RulebookArgs& a, const ListsWork& lw, int32_t max_words, hipStream_t st);
// Clears both alternating input bitmaps (nwords each) and the four error /
// counter words: once per bound workspace, before its first build.
hipError_t launch_rulebook_reset(uint64_t* bits_a, uint64_t* bits_b, int64_t nwords, int32_t* err, hipStream_t st);

// ---------------------------------------------------------------------------
// gather GEMM: out[m][n] = epi( sum_k A(m,k) * Bt[n][k] ),
//   A(m, k) = src[rmap[m*A + f]][c] with k = f*cseg + c   (rmap entry -1: zero;
//   rmap null: source row m, A must be 1)

enum Epilogue : int32_t {
  EPI_BIAS_RELU = 0,   // + bias, ReLU, store in storage dtype
  EPI_BIAS_F32 = 1,    // + bias, store float32
  EPI_F32 = 2,         // store float32
  EPI_STORE = 3,       // store in storage dtype
  EPI_BIAS_LRELU = 4,  // + bias, leaky rectifier (x/3 below zero), store in storage dtype
  EPI_STORE_MASK = 5,  // times act_factor(mask[m][n], slope), store in storage dtype
};

// Arguments of the bias and ground-row sums of one convolution (launch_ground).
struct GroundArgs {
  // pooling layer above (B1 = 0: none)
  const void* dY;
  const uint8_t* argmax;
  const int32_t* Rp;
  const int32_t* n_pool;
  int32_t B1;
  const void* Y_below;  // the convolution's output (ReLU mask of row 0)
  // the pooling layer's output: the routed child's value, so its rectifier
  // derivative (a window's maximum is a copy of the child it came from)
  const void* X_pool;
  // AC == 4: the pooling layer's child ground masks (RulebookArgs::gmask)
  const uint16_t* gmask;
  // the convolution
  void* dZ;            // delta, rows 0..n; row 0 written when B1 > 0
  const int32_t* R;    // its window list [rows][AC]
  const int32_t* n_rows;
  int32_t B2;
  int32_t stride, cp, c_out;
  float slope;  // rectifier of the convolution (0: ReLU, 1/3: leaky)
  float* part;  // [(2 + AC) * cp * PM]
  int32_t PM;   // partial stride, >= B1, B2
  float* db;
  float* D0;
  // > 0: the partials come from the epilogue of the GEMM that wrote dY, one per
  // tile of route_bm pooling rows (rows 1..n_pool): only the first
  // ceil(n_pool / route_bm) of the B1 = B2 are read
  int32_t route_bm;
};

// Row 0 of the gradient below a convolution (its ground row): for input channel
// c, sum over window positions f and outputs n of W[f][c][n] * D0[f][n], times
// the rectifier derivative of the layer below when that layer is a convolution
// (Y_below non-null).
struct Row0Args {
  const void* W;
  const float* D0;
  int32_t A, c_in, c_out, cp_in;
  void* grad_in;
  const void* Y_below;
  float slope;
};

// Work that rides along as extra workgroups at the end of another launch (the
// last `blocks` workgroups of the grid), independent of that launch's own work:
//   kind 1: the ground final pass of a convolution (one workgroup per channel, cp);
//   kind 2: row 0 of the gradient below a convolution (one per channel, cp_in);
//   kind 3: kind 1 below a pooling layer whose row 0 gradient (kind 2 of the
//           convolution above it, r) is computed first, in the same workgroup.
struct ExtraTask {
  int32_t kind;    // 0: none
  int32_t blocks;
  int32_t AC;      // kind 1: window positions whose ground sums are finished (0..9)
  GroundArgs g;
  Row0Args r;
};

struct GemmArgs {
  const void* src;
  int32_t src_stride;
  const int32_t* rmap;
  int32_t A;
  int32_t cseg;
  int32_t K;
  int32_t Kpad;
  const void* Bt;
  int32_t Npad;
  const float* bias;
  int32_t N;
  int32_t out_cols;
  void* out;
  int32_t out_stride;
  int32_t epi;
  const int32_t* rows_dev;  // rows = *rows_dev + rows_add when set, else rows_host
  int32_t rows_add;
  int32_t rows_host;
  int32_t row_begin;
  int32_t cfg;        // tile shape (see plan_gemm)
  int32_t sk;         // GEMM_DIRECT: waves per workgroup, each summing one K range
  int32_t ksplit;     // > 1: K split over workgroups, fp32 partials in part
  float* part;        // [ksplit][part_rows][Npad]
  int32_t part_rows;  // row capacity of part
  // EPI_STORE_MASK: the rectifier derivative of the layer below, from its
  // stored output [rows][mask_stride] (same rows and columns as out)
  const void* mask;
  int32_t mask_stride;
  float slope;
  // optional timing events (timing-enabled events, or null): t_start is recorded
  // when the GEMM kernel starts, t_stop when the last kernel of the launch
  // (the GEMM, or its split-K reduce) ends
  hipEvent_t t_start, t_stop;
  ExtraTask x;  // extra workgroups appended to the launch (kind 0: none)
  int32_t partials_only;  // ksplit > 1: leave the fp32 partials, no reduce launch
  // Pooling backward in the epilogue (route = 1; EPI_STORE, ksplit == 1, a
  // tile shape that stages its output): the output rows m >= 1 are the gradient
  // of a pooling layer, routed through its windows to the convolution below
  // (delta rows >= 1, rectifier derivative applied) with that convolution's slot
  // partial sums, one partial per row tile; pr describes both layers (its dY
  // field is unused) and route_ac is the convolution's finished window count
  // (0 or 4).
  int32_t route;
  int32_t route_ac;
  GroundArgs pr;
  // Pooling forward in the epilogue (pool_fwd = 1; a convolution with the
  // bias-rectifier epilogue, ksplit == 1, a tile shape that stages its output):
  // the GEMM rows are the slots 4 p + f of the pooling windows, rows = 4 (n_pool
  // + 1) from rows_dev / rows_add (the pooling layer's count); slot q computes
  // the convolution row pslot[q] (the pooling layer's window list; row 0 for an
  // inactive location, which then gives the ground value) and stores it (row 0
  // from slot 0 only), and each window's first maximum goes to pool_out /
  // pool_argmax (row stride pool_stride).
  int32_t pool_fwd;
  const int32_t* pslot;
  void* pool_out;
  uint8_t* pool_argmax;
  int32_t pool_stride;
  // set by launch_gemm: the row bound the grid is sized for (rows, or slots with
  // pool_fwd); every window list and row buffer a launch reads holds that many
  // rows, so loads below it may be issued before the device-side count arrives
  int32_t rows_cap;
};

// Template value of the gather GEMMs for the pooling-forward epilogue (the
// others: -1 plain, -3 the masked store EPI_STORE_MASK, 0 or 4 the pooling
// backward with that window count).
constexpr int POOL_FWD_MODE = -2;
constexpr int MASK_MODE = -3;

// Byte range of the buffer descriptor through which the bf16 gather GEMM reads
// its source rows; offsets at or past it read zero (rows without a window
// entry use that), so every source row must end below it.
constexpr uint32_t GATHER_SRC_BYTES = 0x7ffffff0u;

// Whether a tile shape stages its output tile through LDS (16-byte stores), as
// the pooling backward in the epilogue needs.
bool gemm_routes(bool bf16, int cfg);
// Row tile height of a tile shape.
int gemm_bm(bool bf16, int cfg);

// Tile shape and padding of one GEMM, chosen on the host from its row bound.
struct GemmPlan {
  int cfg = 3;
  int BN = 64;
  int Npad = 0;
  int Kpad = 0;
  int ksplit = 1;
  int sk = 1;  // direct kernel (cfg = GEMM_DIRECT): waves per workgroup splitting K
};

// cfg value of the bf16 direct-operand kernel (gemm_direct.hip): 32 x 64 output
// tiles, each wave loading its MFMA operands straight from memory
constexpr int GEMM_DIRECT = 4;
constexpr int DIRECT_BM = 32, DIRECT_BN = 64;

// weight-gradient GEMM, split over sites:
//   part[chunk][m][n] = sum_{o in chunk} A(o, m) * dsrc[o][n]
//   A(o, m) = src[rmap[o*A + f]][c] for m = f*cseg + c < A*cseg;
//   A(o, m_ones) = 1 when m_ones >= 0 (row m_ones of the result is then db)
struct WGradArgs {
  const void* src;
  int32_t src_stride;
  const int32_t* rmap;
  int32_t A;
  int32_t cseg;
  int32_t m_ones;
  int32_t Mpad;
  const void* dsrc;
  int32_t dsrc_stride;
  int32_t dsrc_cols;
  int32_t Npad;
  const int32_t* rows_dev;
  int32_t rows_add;
  int32_t rows_host;
  int32_t nchunks;  // planned (most) site chunks; partials hold that many
  int32_t slabs;    // slabs of sites per chunk: chunks = min(nchunks, rows / (slabs * BK))
  float* part;
  int32_t cfg;  // 0: 128 x 128 tiles, 1: 128 x 64 tiles
  // with nchunks == 1 the kernel writes the results itself (no partials):
  float* dW;  // [A*c_in x c_out]
  float* db;  // [c_out]
  int32_t c_in, c_out;
};

// Weight gradients of several layers in one launch (all with the same tile).
constexpr int MAX_WG_LAYERS = 20;  // convolutions (<= 2*ell + 2) + softmax layer
struct WGradGroup {
  int32_t n;
  int32_t tile_beg[MAX_WG_LAYERS + 1];  // workgroup tiles of layer l: [tile_beg[l], tile_beg[l+1])
  int32_t blk_beg[MAX_WG_LAYERS + 1];   // reduce blocks of layer l
  int32_t G[MAX_WG_LAYERS];             // reduce thread groups of layer l
  int32_t BK;                           // sites per slab
  WGradArgs L[MAX_WG_LAYERS];
};

struct GemmTile {
  int BM, BN, BK;
};
GemmTile gemm_tile(bool bf16, int cfg);
GemmPlan plan_gemm(bool bf16, int64_t max_rows, int N, int K, bool short_rows, int direct_max);
// weight-gradient tiles: 128 rows of dW, 128 or 64 columns
constexpr int WG_BM = 128;
inline int wgrad_bn(int c_out) { return (c_out + 127) / 128 * 128 <= (c_out + 63) / 64 * 64 ? 128 : 64; }

hipError_t launch_gemm(bool bf16, const GemmArgs& a, int64_t max_rows, hipStream_t st);
hipError_t launch_gemm_direct(const GemmArgs& a, int64_t max_rows, hipStream_t st);
// Convolution forward on the vector ALUs for layers with few input channels:
// at most NARROW_KMAX products per output (A * cin, 1 <= cin <= 4, within one
// 16-byte vector of input channels), a window list, the bias-rectifier epilogue,
// optionally the pooling forward above (GemmArgs::pool_fwd, max_rows then counting the
// slots).  conv_narrow_ok tells whether a launch qualifies.
constexpr int NARROW_KMAX = 32;
bool conv_narrow_ok(bool bf16, const GemmArgs& a, int cin);
hipError_t launch_conv_narrow(bool bf16, const GemmArgs& a, int cin, int64_t max_rows, hipStream_t st);
// Weight gradients of n layers that all use tile shape cfg (0: 128 x 128,
// 1: 128 x 64) in one launch.
// extra: a ground final pass (ExtraTask kind 1 or 3) riding on the launch; it
// must not write what the launch's layers read.
hipError_t launch_wgrad(bool bf16, int cfg, const WGradArgs* layers, int n, hipStream_t st,
                        const ExtraTask* extra = nullptr);

// part -> dW [A*c_in x c_out] (and db [c_out] when m_ones >= 0) for every layer
// of the list with nchunks > 1, in one launch.
hipError_t launch_wgrad_reduce(bool bf16, const WGradArgs* layers, int n, hipStream_t st);
// grad_in[0][c] = sum_f sum_n W[(f*c_in + c)*c_out + n] * D0[f][n], times
// act_factor(Y_below[0][c], slope) when Y_below (the layer below's stored
// output, a convolution) is given
hipError_t launch_row0_dx(bool bf16, const void* W, const float* D0, int32_t A, int32_t c_in, int32_t c_out,
                          int32_t cp_in, void* grad_in, const void* Y_below, float slope, hipStream_t st);

// ---------------------------------------------------------------------------
// max-pooling

hipError_t launch_pool_fwd(bool bf16, const void* X_in, int32_t stride_in, const int32_t* R, void* X_out,
                           int32_t stride_out, uint8_t* argmax, int32_t cp, const int32_t* n_out, int64_t cap_out,
                           hipStream_t st);
// Bias gradient db [c_out] and ground-row sums D0 [AC x c_out] (AC in {0, 1, 4,
// 9}) of a convolution with output gradient delta = dZ, and, with a pooling
// layer above (B1 > 0), row 0 of delta itself.  Needs delta rows >= 1 and, with
// a pooling layer, that layer's dY (rows 0..n_pool), argmax and windows Rp.
// kind 0: partial sums over delta rows >= 1 (and, with B1 > 0, over the pooling
//         rows), then the final pass;
// kind 1: pooling backward fused with those partial sums (writes delta rows >= 1;
//         needs B1 == B2);
// kind 2: the final pass alone, over partials written by kind 1 or 3;
// kind 3: the partial sums of kind 0 alone.
// extra: work appended as extra workgroups of the first kernel launched.
hipError_t launch_ground(bool bf16, const GroundArgs& g, int32_t AC, int kind, hipStream_t st,
                         const ExtraTask* extra = nullptr);
// the extra task alone, as its own launch
hipError_t launch_extra(bool bf16, const ExtraTask& x, hipStream_t st);

// ---------------------------------------------------------------------------
// input, parameters, head

hipError_t launch_scatter_input(bool bf16, const void* feats, int32_t n, int32_t c_in, const int32_t* perm, void* X0,
                                int32_t cp0, hipStream_t st);
hipError_t launch_gather_dfeats(bool bf16, const void* grad0, int32_t cp0, const int32_t* perm, int32_t n,
                                int32_t c_in, void* dfeats, hipStream_t st);
// One packing of a weight matrix into a GEMM's [N][K] operand (zero padded):
//   mode 0 (forward):   Bt[n][f*cp_in + c]  = W[(f*c_in + c)*c_out + n]
//   mode 1 (backward):  Bt[c][f*cp_out + n] = W[(f*c_in + c)*c_out + n]
struct PackJob {
  const void* W;
  void* Bt;
  int32_t mode, A, c_in, c_out, cp_in, cp_out, Npad, Kpad;
};
// The input scatter (rows of X0 from the caller's feature rows), run as extra
// workgroups of the packing launch: X0[perm[i]] = feats[i], row 0 = 0.
struct ScatterArgs {
  const void* feats;
  int32_t n, c_in;
  const int32_t* perm;
  void* X0;
  int32_t cp0;
  int32_t blocks;  // workgroups given to it (0: no scatter)
};
struct PackArgs {
  int32_t njobs;
  int32_t tile_beg[2 * MAX_LAYERS + 1];  // first tile of each job in the flat tile range (set by the launcher)
  PackJob job[2 * MAX_LAYERS];
  ScatterArgs sc;
};
// All packings of a step (and, with sc.feats or sc.n == 0 and sc.X0 set, the
// input scatter) in one launch.
hipError_t launch_pack_all(bool bf16, const PackArgs& pa, hipStream_t st);
// counter: a zero int32 in device memory; the last workgroup sums the loss terms
// and sets it back to zero
hipError_t launch_softmax_xent(bool bf16, const float* logits, const int32_t* labels, int32_t batch, int32_t classes,
                               void* dlogits, int32_t dl_stride, float* loss_part, float* loss, int32_t* counter,
                               int32_t* err, hipStream_t st);


// dropout.hip: Xd = X with rows 1 .. *n_rows dropped (row 0 copied; X == Xd:
// in place, row 0 untouched); the softmax layer's input hd[b] =
// X_top[head_rows[b]] dropped with row key b
hipError_t launch_dropout_rows(bool bf16, const void* X, void* Xd, int32_t cp, const int32_t* n_rows, int64_t max_rows,
                               const DropArgs& d, hipStream_t st);
hipError_t launch_head_drop(bool bf16, const void* X_top, const int32_t* head_rows, int32_t batch, int32_t cp,
                            void* hd, const DropArgs& d, hipStream_t st);
hipError_t launch_fill_zero(void* p, int64_t bytes, hipStream_t st);

// Backward of the softmax layer's input, fused with the top convolution's
// bias / ground-row sums: dh[b] = sum over splits of dh_part (the softmax-layer
// input-gradient GEMM's split-K partials, or dh itself with ksplit 1), times the
// dropout factor; the top layer's row of sample b gets dh[b] * f'(Y_top); the
// partial sums (head_backward_parts(batch) partials per slot) hold slot 0, the
// sum over empty samples, and slots 1, 2+f as in launch_ground; row 0 of
// grad_top is zeroed so that the final ground pass, run with B1 = B2 = parts,
// dY = Y_below = the top layer, finishes row 0 as below a pooling layer.
struct HeadBwdArgs {
  const float* dh_part;
  int32_t ksplit;
  int64_t ks_stride;  // floats between splits
  int32_t dh_stride;  // floats between samples
  const int32_t* head_rows;
  int32_t batch;
  const void* Y_top;
  void* grad_top;
  int32_t cp;
  float slope;
  DropArgs drop;
  const int32_t* R;  // the top convolution's window list [rows][AC]
  float* part;       // [(2 + AC) * cp * PM]
  int32_t PM;
};
int head_backward_parts(int32_t batch);
hipError_t launch_head_backward(bool bf16, const HeadBwdArgs& h, int32_t AC, hipStream_t st,
                                const ExtraTask* extra = nullptr);

// encode.hip: pen paths -> sites and 9 features (Section 2.4)
struct EncodeArgs {
  const int32_t* points;  // [n_points][2] (y, x)
  const int32_t* begin;   // [n_strokes + 1]
  const int32_t* sample;  // [n_strokes]
  int32_t n_points, n_strokes, batch, N, Wd, max_sites;
  uint64_t* bits;    // [batch][N][Wd] occupancy
  int32_t* wpre;     // [batch][N][Wd] exclusive popcount prefix within the sample
  int32_t* scount;   // [batch]
  int32_t* soff;     // [batch]
  int32_t* total;    // [1] distinct sites
  int32_t* err;      // [1] ERRBIT_*
  int32_t* counts;   // [max_sites][8] move counts
  int32_t* coords;   // [max_sites][3] output
};
hipError_t launch_encode(bool bf16, const EncodeArgs& a, void* feats, hipStream_t st);

// sgd.hip: one momentum-SGD update of many parameter arrays in one launch
constexpr int MAX_SGD_JOBS = 2 * MAX_LAYERS;
struct SgdJob {
  float* w;          // fp32 master
  void* w_store;     // storage-dtype copy to refresh, or null
  const float* g;    // gradient
  float* v;          // velocity
  int64_t n;
  float wd;          // weight decay
};
struct SgdArgs {
  int32_t njobs;
  int32_t store_bf16;
  float lr, momentum;
  int32_t blk_beg[MAX_SGD_JOBS + 1];
  SgdJob job[MAX_SGD_JOBS];
};
hipError_t launch_sgd(const SgdArgs& a, hipStream_t st);

}  // namespace sscn
