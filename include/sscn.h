/*
 * sscn.h -- spatially-sparse DeepCNet forward and backward pass on one AMD
 * Instinct MI355X (gfx950).
 *
 * The calls follow the statement of the problem in Graham, "Spatially-sparse
 * convolutional neural networks" (arXiv:1409.6070): a batch of active sites,
 * each with a feature vector, on an N x N grid (Sections 1, 2.4, 2.5), fed to
 * the layer list of a DeepCNet(ell, k) (Section 2.1):
 *
 *     input - kC3 - MP2 - 2kC2 - MP2 - ... - (ell+1)kC2 - softmax output
 *
 * with N = 3 * 2^ell, valid stride-1 convolutions, 2x2 stride-2 max-pooling,
 * ReLU on hidden layers, or of a DeepCNiN(ell, k) (Section 2.2): the same with
 * a 1x1 convolution (kC1, 2kC1, ...) after every pooling layer and after the
 * last convolution, and the leaky rectifier f(x) = x (x >= 0), x/3 (x < 0) on
 * every hidden layer.  Only active sites are computed; every inactive site of
 * a layer shares that layer's ground state (Section 2.3), kept as row 0 of
 * the layer's feature matrix.
 *
 * Stages, layers and parameters.  DeepCNet has L = 2*ell + 1 stages, DeepCNiN
 * L = 3*ell + 2; layer 0 is the input and layer s = 1 .. L the output of stage s.
 * The convolutions, counted in stage order, own weight matrices
 * n = 0 .. n_conv - 1 (n_conv = ell + 1, or 2*ell + 2 for DeepCNiN); the
 * softmax layer's matrix is n_conv, so there are n_conv + 1 of them.
 *
 * Memory ownership.  The caller owns every device buffer: inputs, parameters,
 * gradients, logits, loss and one workspace.  The library never allocates or
 * frees device memory and never synchronises, except in sscn_layer_sizes().
 * All work is enqueued on the stream passed in (a hipStream_t, NULL for the
 * null stream).  A net is used from one host thread and one stream at a time.
 *
 * Layouts.  Row-major throughout.  Convolution weight n is a [F*F*C_in, C_out]
 * matrix whose row index is (dy*F + dx)*C_in + c (cross-correlation: output
 * (y, x) reads input (y+dy, x+dx)); F = 3 for n = 0, 1 for the 1x1 layers, else
 * 2.  The softmax layer's matrix is [C_last, n_classes].
 * Weights and input features are in the net's storage dtype; biases, weight
 * and bias gradients, logits and the loss are float32.
 *
 * Errors.  Argument errors are returned at once.  Data errors found on the
 * device (a site outside the grid or batch, a site listed twice) are latched
 * in the workspace and returned by the next sscn_layer_sizes(); results
 * computed from such input are undefined but every kernel stays within its
 * buffers.  No C++ exception crosses this interface and nothing exits the
 * process.
 */
#ifndef SSCN_H
#define SSCN_H

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__) || defined(__clang__)
#define SSCN_API __attribute__((visibility("default")))
#else
#define SSCN_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SSCN_OK = 0,
  SSCN_ERR_INVALID_ARGUMENT = 1, /* null pointer, bad size or index          */
  SSCN_ERR_OUT_OF_RANGE = 2,     /* a site outside [0,batch) x [0,N)^2        */
  SSCN_ERR_DUPLICATE_SITE = 3,   /* the same (b, y, x) listed twice           */
  SSCN_ERR_CAPACITY = 4,         /* n > max_active or batch > batch_max       */
  SSCN_ERR_BAD_STATE = 5,        /* call out of order (e.g. forward before build) */
  SSCN_ERR_HIP = 6,              /* a HIP runtime call failed                 */
  SSCN_ERR_WORKSPACE = 7         /* workspace null, too small or misaligned   */
} sscn_status;

typedef enum { SSCN_F32 = 0, SSCN_BF16 = 1 } sscn_dtype;

/* Network family (Sections 2.1, 2.2). */
typedef enum {
  SSCN_DEEPCNET = 0, /* DeepCNet(ell, k): conv3, then (2x2 max-pool, conv2) x ell; ReLU          */
  SSCN_DEEPCNIN = 1  /* DeepCNiN(ell, k): DeepCNet plus a 1x1 convolution (same width) after every
                        pooling layer and after the last convolution; leaky rectifier x/3 below 0 */
} sscn_arch;

/* A DeepCNet(ell, k) or DeepCNiN(ell, k) (arch) with c_in input features per
 * site and an n_classes softmax output (Sections 2.1, 2.2).  batch_max and
 * max_active bound the batches that sscn_rulebook_build accepts and size the
 * workspace.  dtype is the storage type of features, weights and stored
 * activations/gradients; products and sums accumulate in float32. */
typedef struct {
  int32_t ell;
  int32_t k;
  int32_t c_in;
  int32_t n_classes;
  int32_t batch_max;
  int32_t max_active;
  int32_t dtype;   /* sscn_dtype */
  int32_t arch;    /* sscn_arch */
  int32_t dropout; /* nonzero: the workspace also holds the dropped copies of every
                      dropout level's input, so sscn_set_dropout may set rates > 0 */
} sscn_net_desc;

typedef struct sscn_net sscn_net; /* opaque host-side plan */

/* One layer of the network as stored in the workspace (for tests and
 * inspection).  Layer 0 is the input; layer s = 1 .. L is the output of
 * stage s (a convolution or a pooling layer, see kind).  All pointers are device
 * pointers into the workspace bound by the last sscn_rulebook_build. */
typedef struct {
  int32_t kind;       /* 0 input, 1 convolution, 2 max-pooling                  */
  int32_t side;       /* spatial side S of the layer                            */
  int32_t channels;   /* C: features per site                                   */
  int32_t row_stride; /* elements per feature/gradient row (C rounded up)       */
  int32_t window;     /* A = F*F positions per window (0 for the input layer)   */
  int32_t capacity;   /* rows available for active sites (ground row excluded)  */
  const int32_t* count;  /* [1] number n of active sites, set by rulebook_build  */
  const int32_t* sites;  /* [capacity] rows 1..n: key (b*S + y)*S + x, ascending */
  const int32_t* rules;  /* [(capacity+1) * A]: row of the layer below read by
                            window position (dy*F + dx) of each row; 0 = ground;
                            row 0 is all 0                                      */
  const int32_t* rules_t;/* convolution: [(capacity_below+1) * A]: for each row
                            i of the layer below, the row whose window holds i at
                            position f, -1 if none.  Pooling: [capacity_below+1]
                            parent row * 4 + position, -1 if none.              */
  void* features;        /* [(capacity+1) * row_stride] storage dtype, row 0 = ground */
  void* grad;            /* same shape: convolution dL/dZ (pre-activation),
                            pooling and input dL/dX; row 0 = sum over inactive sites */
  uint8_t* argmax;       /* pooling: [(capacity+1) * row_stride] window position
                            (0..3, first maximum in (dy, dx) order) of each max  */
  const uint16_t* gmask; /* pooling layer on a 2x2 convolution (else NULL):
                            [capacity+1] per row, bit 4 f + k set when window
                            position k of the convolution row at pooling position
                            f reads an inactive location (the ground row) of the
                            layer below that convolution; row 0 all set.  Used by
                            the pooling backward for the ground-row sums.       */
} sscn_layer_view;

/* Host only.  Validates desc (ell in 1..8, k, c_in, n_classes, batch_max,
 * max_active >= 1, dtype and arch known) and builds the plan. */
SSCN_API sscn_status sscn_net_create(const sscn_net_desc* desc, sscn_net** out);
SSCN_API void sscn_net_destroy(sscn_net* net);
SSCN_API const char* sscn_status_string(int32_t status);

/* Number of parameter matrices (n_conv + 1) and the shape of matrix `layer`
 * (0 .. ell convolutions, ell+1 softmax layer); the bias has `cols` entries.
 * Section 2.1 gives the weight count 3^2*M*k + sum_n 2^2*(n k)*((n+1) k). */
SSCN_API int32_t sscn_net_num_params(const sscn_net* net);
SSCN_API sscn_status sscn_net_param_shape(const sscn_net* net, int32_t layer, int64_t* rows, int64_t* cols);

/* Bytes of device workspace the net needs (an upper bound for any batch
 * within batch_max / max_active).  The workspace must be 256-byte aligned
 * and left untouched from sscn_rulebook_build through sscn_backward. */
SSCN_API sscn_status sscn_net_workspace_bytes(const sscn_net* net, size_t* bytes);

/* Builds every layer's active-site set and window lists (Section 2.3: the
 * pointer matrix, here a rank-indexed occupancy bitmap per layer) for
 * d_coords[n][3] = (b, y, x), int32, any order, 0 <= b < batch, 0 <= y,x < N.
 * Rows are numbered in ascending (b, y, x) order.  Asynchronous; device-side
 * input errors are reported by sscn_layer_sizes. */
SSCN_API sscn_status sscn_rulebook_build(sscn_net* net, const int32_t* d_coords, int32_t n, int32_t batch,
                                void* d_workspace, size_t workspace_bytes, void* stream);

/* sscn_rulebook_build for sites grouped by sample (Section 2.3 builds each
 * sample's pointer matrices from that sample's input alone): d_sample_begin
 * is a device array of batch + 1 int32, non-decreasing, d_sample_begin[0] = 0,
 * d_sample_begin[batch] = n, and sample b's sites are rows
 * d_sample_begin[b] .. d_sample_begin[b + 1] - 1 of d_coords, each with b in
 * its first column (any order within the sample).  The result is the same as
 * sscn_rulebook_build's on the same sites; the bitmap pass inserts each
 * sample's sites itself, so no insertion launch precedes it.  A site outside
 * its sample's range or the grid, inconsistent offsets (read with every
 * index clamped to 0 .. n) and duplicate sites are device-side input errors
 * (SSCN_ERR_OUT_OF_RANGE, SSCN_ERR_DUPLICATE_SITE from sscn_layer_sizes);
 * argument errors as for sscn_rulebook_build, and d_sample_begin null. */
SSCN_API sscn_status sscn_rulebook_build_grouped(sscn_net* net, const int32_t* d_coords, const int32_t* d_sample_begin,
                                                 int32_t n, int32_t batch, void* d_workspace, size_t workspace_bytes,
                                                 void* stream);

/* Synchronises `stream`, copies the L + 1 active-site counts (layer 0 =
 * input, then each stage) to h_counts, and returns any latched input error
 * (SSCN_ERR_OUT_OF_RANGE / SSCN_ERR_DUPLICATE_SITE).  It also returns
 * SSCN_ERR_OUT_OF_RANGE, once, when a training sscn_forward since the last such
 * report met a label outside [0, n_classes) (counts are still written). */
SSCN_API sscn_status sscn_layer_sizes(sscn_net* net, int32_t* h_counts, void* stream);

/* Forward pass (Sections 2.1, 2.3): d_feats[n][c_in] (storage dtype, in the
 * order given to sscn_rulebook_build); h_W / h_b host arrays of n_conv + 1 device
 * pointers (weights in storage dtype, biases float32); d_labels[batch] int32
 * in [0, n_classes).  Writes d_logits[batch][n_classes] and *d_loss (mean
 * softmax cross-entropy), both float32.  A label outside [0, n_classes) is
 * latched on the device (the next sscn_layer_sizes returns
 * SSCN_ERR_OUT_OF_RANGE); that sample's loss term and one-hot term are 0.  With d_labels and d_loss both null
 * the pass is inference only: it writes the logits, skips the loss and the
 * backward-only work, and a following sscn_backward returns
 * SSCN_ERR_BAD_STATE.  Exactly one of them null: SSCN_ERR_INVALID_ARGUMENT. */
SSCN_API sscn_status sscn_forward(sscn_net* net, const void* d_feats, const void* const* h_W, const float* const* h_b,
                         const int32_t* d_labels, float* d_logits, float* d_loss, void* stream);

/* Backward pass of the last sscn_forward (Section 2.3: the same structures in
 * reverse).  h_dW / h_db: host arrays of n_conv + 1 device float32 pointers shaped
 * like the parameters; they are overwritten (not accumulated).  d_dfeats
 * (nullable): [n][c_in] storage dtype, gradient of the loss with respect to
 * the input features, in the caller's site order. */
SSCN_API sscn_status sscn_backward(sscn_net* net, float* const* h_dW, float* const* h_db, void* d_dfeats, void* stream);

/* Dropout per level (Section 2.1), applied by every following training pass
 * (sscn_forward with labels, and its sscn_backward); inference passes ignore it.
 * h_rates[n_rates] (host, n_rates = ell + 2): the rate for the input of each
 * convolution that is not 1x1, in stage order (ell + 1 of them; Section 2.2
 * applies no dropout to the 1x1 network-in-network layers), then the rate for
 * the softmax layer's input; each in [0, 1).  n_rates = 0 (h_rates may be null)
 * switches dropout off.  seed: the 64-bit key of the masks.
 *
 * Inverted dropout: a kept value is multiplied by 1/(1 - p) (a float32 value),
 * a dropped one becomes 0; the backward pass applies the same factors.  Only
 * rows 1.. (active sites) of a level's input are dropped: the ground row, the
 * state shared by all inactive sites, passes unchanged.  Element (channel c)
 * of the row with key q of level j is kept when word c % 4 of
 * sscn_philox4x32_10(counter = {q, c / 4, j, 0}, key = {seed mod 2^32,
 * seed / 2^32}) is >= floor(p * 2^32); q is the site key (b*S + y)*S + x of
 * the level's input layer, or the sample index b for the softmax input.
 * Rates > 0 need a net created with desc.dropout != 0, else
 * SSCN_ERR_INVALID_ARGUMENT; so does a wrong n_rates or a rate outside [0, 1).
 * A successful call also ends the current pass: sscn_backward then returns
 * SSCN_ERR_BAD_STATE until the next training sscn_forward. */
SSCN_API sscn_status sscn_set_dropout(sscn_net* net, const double* h_rates, int32_t n_rates, uint64_t seed);

/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC 2011), the generator of the
 * dropout masks, evaluated on the host: out = the four output words for the
 * four-word counter and two-word key (host arrays).  For reproducing masks. */
SSCN_API void sscn_philox4x32_10(const uint32_t counter[4], const uint32_t key[2], uint32_t out[4]);

/* One stochastic-gradient-descent update of every parameter from the gradients
 * of the last sscn_backward (the dW / db arrays passed to it, which must still
 * hold them).  Host arrays of n_conv + 1 device pointers:
 *   h_W32  float32 master weights [rows][cols] (updated in place)
 *   h_W    the storage-dtype weights the next sscn_forward reads, rewritten from
 *          the updated masters (required for bf16 nets; for float32 nets it may
 *          be null or equal to h_W32, and the masters are then those weights)
 *   h_b    float32 biases (updated in place)
 *   h_vW, h_vb  float32 velocities shaped like the weights and biases (zero
 *          them before the first step)
 * Classical momentum with L2 weight decay on the weights only (the optimiser is
 * not stated in the paper; this is the usual library convention):
 *   g = dW + weight_decay * W (biases: g = db);  v = momentum * v + g;
 *   W = W - lr * v.
 * lr, momentum and weight_decay must be finite and >= 0.  Returns
 * SSCN_ERR_BAD_STATE unless sscn_backward has run since the last forward or
 * build.  One launch; asynchronous. */
SSCN_API sscn_status sscn_sgd_step(sscn_net* net, float* const* h_W32, void* const* h_W, float* const* h_b,
                                   float* const* h_vW, float* const* h_vb, float lr, float momentum,
                                   float weight_decay, void* stream);

/* Online pen strokes -> sparse input with M = 9 features (Section 2.4): per
 * grid square the picture of the pen's path (feature 0, 1 where the pen went)
 * and an 8-bin histogram of its movement in the compass directions E, NE, N,
 * NW, W, SW, S, SE (features 1..8; counter-clockwise, north = -y).
 *
 * d_points[n_points][2]: (y, x) int32 grid points, 0 <= y, x < N, all strokes
 * concatenated; stroke s is points d_stroke_begin[s] .. d_stroke_begin[s+1]-1
 * (d_stroke_begin has n_strokes + 1 entries, from 0 to n_points,
 * non-decreasing) and belongs to sample d_stroke_sample[s] in [0, batch).
 * Consecutive points p0, p1 of a stroke are joined by the pixels
 * p0 + round_half_up(i * (p1 - p0) / L), i = 0 .. L, L = max(|dy|, |dx|)
 * (an 8-connected line).  Each unit move between consecutive pixels gives half
 * its length (1, or sqrt 2 for a diagonal) to its direction's feature at both
 * squares it joins.  Sites: every touched square, ascending (b, y, x).
 *
 * Writes d_coords[n][3] (b, y, x) and d_feats[n][9] (dtype: sscn_dtype) for
 * the n distinct sites, *h_count = n, and synchronises `stream`.  Returns
 * SSCN_ERR_CAPACITY when n > max_sites (*h_count still set; the first
 * max_sites sites written), SSCN_ERR_OUT_OF_RANGE for a point outside the grid
 * or a sample outside the batch, SSCN_ERR_INVALID_ARGUMENT for bad offsets.
 * d_ws: device scratch of sscn_encode_workspace_bytes(N, batch, max_sites)
 * bytes, 256-byte aligned, free for other use between calls. */
SSCN_API sscn_status sscn_encode_workspace_bytes(int32_t N, int32_t batch_max, int32_t max_sites, size_t* bytes);
SSCN_API sscn_status sscn_encode_strokes(int32_t N, int32_t dtype, const int32_t* d_points, int32_t n_points,
                                         const int32_t* d_stroke_begin, const int32_t* d_stroke_sample,
                                         int32_t n_strokes, int32_t batch, int32_t* d_coords, void* d_feats,
                                         int32_t max_sites, int32_t* h_count, void* d_ws, size_t ws_bytes,
                                         void* stream);

/* sscn_encode_strokes for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same arguments and results without d_ws / ws_bytes.  Its
 * scratch is a fixed array of SSCN_ENCODE_STATIC_SCRATCH_BYTES in device memory
 * that every GPU the library runs on holds until the process ends; the call
 * itself allocates and frees nothing.  It returns SSCN_ERR_WORKSPACE when
 * sscn_encode_workspace_bytes(N, batch, max_sites) exceeds that size, and
 * SSCN_ERR_HIP if the scratch's device address cannot be obtained.  All calls on
 * one GPU share its scratch: calls that overlap on one GPU (concurrent streams
 * or host threads) race and must be serialised by the caller. */
#define SSCN_ENCODE_STATIC_SCRATCH_BYTES ((size_t)16 << 20)
SSCN_API sscn_status sscn_encode_strokes_static(int32_t N, int32_t dtype, const int32_t* d_points, int32_t n_points,
                                                const int32_t* d_stroke_begin, const int32_t* d_stroke_sample,
                                                int32_t n_strokes, int32_t batch, int32_t* d_coords, void* d_feats,
                                                int32_t max_sites, int32_t* h_count, void* stream);

/* Runs only stage s (1 .. L) of the forward or backward pass on the
 * current workspace contents, with the parameters of the last sscn_forward /
 * sscn_backward.  For checking one kernel group against known inputs.  A
 * backward convolution stage takes its output gradient (all rows) as it
 * stands and writes its parameter gradients and the whole gradient below; a
 * backward pooling stage writes the whole gradient below (and, as a side
 * effect, the bias gradient of the convolution below it and row 0 of that
 * convolution's input gradient). */
SSCN_API sscn_status sscn_forward_stage(sscn_net* net, int32_t stage, void* stream);
SSCN_API sscn_status sscn_backward_stage(sscn_net* net, int32_t stage, void* stream);

/* Kernel timing with HIP events, for measurement tools.  Kernel classes: */
typedef enum {
  SSCN_KC_RULEBOOK = 0,   /* active sets, window lists, transposes            */
  SSCN_KC_GATHER_GEMM = 1,/* implicit-gather MFMA GEMM: conv forward, conv input
                             gradient, softmax layer forward and dh          */
  SSCN_KC_WGRAD = 2,      /* split-K MFMA weight gradient                      */
  SSCN_KC_WGRAD_REDUCE = 3,/* split-K partial sums -> dW (and the softmax db)  */
  SSCN_KC_POOL_FWD = 4,
  SSCN_KC_POOL_BWD = 5,   /* routing through the windows, with the ground-row,
                             bias and ground-window sums of the conv below    */
  SSCN_KC_HEAD = 6,       /* input scatter, weight packing, softmax, loss, scatter of dh */
  SSCN_KC_GROUND = 7,     /* bias and ground-window sums of a conv not under a
                             pooling layer; ground-row input gradient        */
  SSCN_KC_DROPOUT = 8,    /* dropped copies of the dropout levels' inputs      */
  SSCN_KC_SGD = 9,        /* the parameter update of sscn_sgd_step             */
  SSCN_KC_CONV_NARROW = 10,/* convolution forward with few input channels (at most
                             32 products per output, e.g. the first layer of a
                             one-channel input) on the vector ALUs, with the
                             pooling forward above it                        */
  SSCN_KC_COUNT = 11
} sscn_kernel_class;

/* While enabled, every launch of a kernel whose class bit (1 << class) is set
 * in class_mask is bracketed by a pair of HIP events recorded on the caller's
 * stream.  A mask of 0 disables timing.  Events are created on first use and
 * destroyed with the net; at most 65536 launches are recorded between two
 * sscn_timing_collect calls (further launches are not timed). */
SSCN_API sscn_status sscn_timing_enable(sscn_net* net, uint32_t class_mask);

/* Synchronises `stream`, then for kernel class `kernel_class` returns the
 * number of timed launches and the sum of their event-measured durations
 * (milliseconds) since the previous collect, and forgets those records. */
SSCN_API sscn_status sscn_timing_collect(sscn_net* net, int32_t kernel_class, int32_t* launches, float* total_ms,
                                         void* stream);

/* Launch roles and plans in the tags of sscn_timing_launches. */
typedef enum {
  SSCN_ROLE_FORWARD = 0,     /* a convolution's forward (with a fused pooling forward: pooled bit) */
  SSCN_ROLE_INPUT_GRAD = 1,  /* a convolution's input gradient (with a fused pooling backward: routed bit) */
  SSCN_ROLE_SOFTMAX_FWD = 2, /* the softmax layer's logits GEMM                                    */
  SSCN_ROLE_SOFTMAX_DH = 3,  /* the softmax layer's input-gradient GEMM                            */
  SSCN_ROLE_OTHER = 4        /* any other launch                                                  */
} sscn_launch_role;
enum { SSCN_PLAN_NONE = 15 }; /* plan field of a launch that is not a gather GEMM */

/* Like sscn_timing_collect, but per launch: synchronises `stream`, writes the
 * first min(capacity, count) timed launches of `kernel_class` since the
 * previous collect, in launch order, as h_tags[i] and h_ms[i] (event-measured
 * duration, milliseconds), sets *count to the number recorded, and forgets
 * them.  tag = stage | role << 8 | plan << 12 | routed << 16 | pooled << 17:
 * stage (bits 0-7) the stage the launch serves (1 .. L; 0 for the softmax
 * layer and other launches), role (bits 8-11) an sscn_launch_role, plan
 * (bits 12-15) the gather-GEMM tile plan (0: 128 x 128, 1: 128 x 64, 2: 64 x 64,
 * 3: 32 x 64 LDS-tiled tiles, 4: the direct-operand 32 x 64 kernel) or
 * SSCN_PLAN_NONE, routed (bit 16) an input gradient that runs the pooling
 * backward below it in its epilogue, pooled (bit 17) a forward that runs the
 * pooling layer above it in its epilogue.  Host arrays; capacity 0 (null
 * arrays) just counts and forgets. */
SSCN_API sscn_status sscn_timing_launches(sscn_net* net, int32_t kernel_class, int32_t* h_tags, float* h_ms,
                                          int32_t capacity, int32_t* count, void* stream);

/* Describes layer `layer` (0 .. L) of the bound workspace. */
SSCN_API sscn_status sscn_layer_view_get(const sscn_net* net, int32_t layer, sscn_layer_view* out);

#ifdef __cplusplus
}
#endif

#endif /* SSCN_H */
