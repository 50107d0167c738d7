// C interface of libsscn: plan, workspace layout and launch sequencing for the
// spatially-sparse DeepCNet forward and backward pass (arXiv:1409.6070,
// Sections 2.1 and 2.3).  Host code only; every kernel is enqueued on the
// caller's stream and no call synchronises except sscn_layer_sizes().

#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "sscn.h"
#include "common.h"
#include "kernels.h"

// site slabs (64 sites) per weight-gradient chunk, 128- and 64-wide tiles
#ifndef WG_SLABS_128
#define WG_SLABS_128 8
#define WG_SLABS_64 12
#endif

using namespace sscn;

namespace {

struct LayerPlan {
  int kind;  // 0 input, 1 conv, 2 pool
  int S, C, Cp, F, A, Wd;
  int64_t cap;
  int conv_index;  // convolution layers: parameter index
  int drop_level;  // convolutions that are not 1x1: dropout level of their input, else -1
  // workspace pointers
  uint64_t* bits;
  int32_t* wpre;
  int32_t* scount;
  int32_t* soff;
  int32_t* sites;
  void* X;
  void* grad;
  int32_t* rules;
  int32_t* rules_t;
  uint8_t* argmax;
  uint16_t* gmask;  // pooling layer on a 2x2 convolution: child ground masks (RulebookArgs::gmask)
  void* Xd;  // dropped copy of X when this layer feeds a dropout level (dropout workspace only)
};

struct ParamPlan {
  int A, c_in, c_out, cp_in, cp_out;  // FC: A = 1, cp_in = Cp_last, cp_out = dlogits stride
  GemmPlan pf, pd;                    // forward (logits) and input-gradient (dh) GEMMs
  int64_t rows_f, rows_d;             // their row bounds
  int NpadF, KpadF, NpadD, KpadD;
  int Mpad_w, Npad_w, bn_w, nchunks, m_ones;
  size_t part_off;  // this layer's split-K partials in wpart (floats)
  void* WpF;
  void* WpD;
};

struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base((char*)b) {}
  void* take(size_t bytes) {
    off = (off + 255) / 256 * 256;
    void* p = base ? base + off : nullptr;
    off += bytes;
    return p;
  }
};

}  // namespace

struct sscn_net {
  sscn_net_desc d;
  bool bf16;
  int esz, VE;
  int nlayers;
  int nparams;
  int nconv;    // convolutional layers (weights 0 .. nconv-1; the softmax layer's is nconv)
  bool nin;     // DeepCNiN (1x1 layers, leaky rectifier)
  float slope;  // negative-side slope of the hidden layers' rectifier
  LayerPlan L[MAX_LAYERS];
  ParamPlan P[MAX_LAYERS];
  int dl_stride;  // dlogits row stride (elements)
  int pool_parts;
  int wgrad_slabs[2];  // slabs of sites per weight-gradient chunk, 128- and 64-wide tiles
  // global workspace pointers
  int32_t* counts;
  int32_t* err;   // [4]: the input-error word, then completion counters (zeroed by every rulebook build,
                  // returned to zero by the kernel that uses them): [1] softmax loss
  int32_t* perm;
  int32_t* head_rows;
  void* dlogits;
  float* dh;
  float* loss_part;
  float* wpart;
  float* gpart;  // split-K partials of the gather GEMMs
  float* D0;
  float* ppart;
  size_t ppart_half;  // floats per convolution-parity half of ppart
  uint64_t* bits0_alt;  // the second input bitmap (builds alternate with L[0].bits)
  int32_t rb_parity;    // which input bitmap and error word the next build uses
  int32_t* err_cur;     // the last build's error word
  size_t d0_half;     // and of D0
  void* hdrop;  // the softmax layer's dropped input [batch_max][Cp_top] (dropout workspace only)
  size_t ws_bytes;
  int32_t max_words;
  // bound state
  void* ws;
  int batch;
  int n;
  bool built, forwarded, backwarded;
  const void* W[MAX_LAYERS];
  const float* b[MAX_LAYERS];
  float* dW[MAX_LAYERS];
  float* db[MAX_LAYERS];
  bool want_dfeats;
  float* logits;
  const int32_t* labels;
  // dropout (Section 2.1): rates per level, set by sscn_set_dropout
  int n_rates = 0;
  double rates[MAX_LAYERS] = {};
  uint64_t seed = 0;
  bool drop_on = false;  // the current pass applies dropout (a training pass with rates set)
  // kernel timing (HIP events around launcher calls of the selected classes)
  uint32_t tmask = 0;
  std::vector<hipEvent_t> ev_pool;
  size_t ev_next = 0;
  struct Rec {
    int cls;
    int32_t tag;  // launch tag (sscn_timing_launches)
    hipEvent_t a, b;
  };
  std::vector<Rec> recs;
  ~sscn_net() {
    for (hipEvent_t e : ev_pool) (void)hipEventDestroy(e);
  }
};

static constexpr size_t MAX_TIMED = 65536;

static hipEvent_t next_event(sscn_net* net) {
  if (net->ev_next == net->ev_pool.size()) {
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    net->ev_pool.push_back(e);
  }
  return net->ev_pool[net->ev_next++];
}

// Runs one launcher call; when its class is being timed, brackets it with two events.
// A gather-GEMM launch; while its class is timed, the kernels themselves record
// the start and end events (the span of the GEMM kernel and its split-K reduce,
// without the dispatch latency that events recorded around the launch include).
// Launch tag of a timed record: stage | role << 8 | plan << 12 | routed << 16 | pooled << 17.
static int32_t launch_tag(int stage, int role, int plan, bool routed = false, bool pooled = false) {
  return (int32_t)(stage & 0xFF) | (role << 8) | (plan << 12) | ((int)routed << 16) | ((int)pooled << 17);
}
static const int32_t TAG_OTHER = launch_tag(0, SSCN_ROLE_OTHER, SSCN_PLAN_NONE);

static hipError_t timed_gemm(sscn_net* net, GemmArgs g, int64_t max_rows, hipStream_t st, int stage, int role) {
  g.t_start = g.t_stop = nullptr;
  hipEvent_t a = nullptr, b = nullptr;
  if ((net->tmask & (1u << SSCN_KC_GATHER_GEMM)) && net->recs.size() < MAX_TIMED && max_rows - g.row_begin > 0) {
    a = next_event(net);
    b = next_event(net);
    if (a && b) {
      g.t_start = a;
      g.t_stop = b;
    }
  }
  const hipError_t e = launch_gemm(net->bf16, g, max_rows, st);
  if (g.t_start && e == hipSuccess)
    net->recs.push_back({SSCN_KC_GATHER_GEMM, launch_tag(stage, role, g.cfg, g.route != 0, g.pool_fwd != 0), a, b});
  return e;
}

template <class F>
static hipError_t timed(sscn_net* net, int cls, hipStream_t st, F&& launch, int32_t tag = TAG_OTHER) {
  if (!(net->tmask & (1u << cls)) || net->recs.size() >= MAX_TIMED) return launch();
  hipEvent_t a = next_event(net), b = next_event(net);
  if (!a || !b) return launch();
  if (hipEventRecord(a, st) != hipSuccess) return hipErrorUnknown;
  hipError_t e = launch();
  if (hipEventRecord(b, st) != hipSuccess) return hipErrorUnknown;
  net->recs.push_back({cls, tag, a, b});
  return e;
}

// Row tiles at capacity (and their height) of the input-gradient GEMM of
// convolution s when it computes the gradient of a pooling layer s-1 on a
// convolution, with a tile shape that can run that layer's backward in its
// epilogue; 0 otherwise.
static int64_t route_tiles(const sscn_net* net, int s, int* bm) {
  if (s < 3) return 0;
  const LayerPlan& L = net->L[s];
  const LayerPlan& Lp = net->L[s - 1];
  if (L.kind != 1 || Lp.kind != 2 || net->L[s - 2].kind != 1 || L.A < 2) return 0;
  const ParamPlan& P = net->P[L.conv_index];
  if (P.pd.ksplit != 1 || !gemm_routes(net->bf16, P.pd.cfg)) return 0;
  *bm = gemm_bm(net->bf16, P.pd.cfg);
  return (Lp.cap + *bm - 1) / *bm;  // rows 1 .. cap
}

static void carve(sscn_net* net, void* base) {
  Carver cv(base);
  const int B = net->d.batch_max;
  net->counts = (int32_t*)cv.take(sizeof(int32_t) * net->nlayers);
  net->err = (int32_t*)cv.take(sizeof(int32_t) * 4);
  net->perm = (int32_t*)cv.take(sizeof(int32_t) * (size_t)net->d.max_active);
  net->head_rows = (int32_t*)cv.take(sizeof(int32_t) * (size_t)B);
  size_t max_part = 0, max_d0 = 0, max_gpart = 0;
  int max_cp = 0;
  for (int s = 0; s < net->nlayers; ++s) {
    LayerPlan& L = net->L[s];
    const size_t words = (size_t)B * L.S * L.Wd;
    L.bits = (uint64_t*)cv.take(words * 8);
    if (s == 0) net->bits0_alt = (uint64_t*)cv.take(words * 8);  // builds alternate input bitmaps
    L.wpre = (int32_t*)cv.take(words * 4);
    L.scount = (int32_t*)cv.take((size_t)B * 4);
    L.soff = (int32_t*)cv.take((size_t)B * 4);
    L.sites = (int32_t*)cv.take((size_t)L.cap * 4);
    L.X = cv.take((size_t)(L.cap + 1) * L.Cp * net->esz);
    L.grad = cv.take((size_t)(L.cap + 1) * L.Cp * net->esz);
    max_cp = std::max(max_cp, L.Cp);
    if (s >= 1) {
      const LayerPlan& Lb = net->L[s - 1];
      L.rules = (int32_t*)cv.take((size_t)(L.cap + 1) * L.A * 4);
      if (L.kind == 1)
        L.rules_t = (int32_t*)cv.take((size_t)(Lb.cap + 1) * L.A * 4);
      else
        L.rules_t = (int32_t*)cv.take((size_t)(Lb.cap + 1) * 4);
      L.argmax = (L.kind == 2) ? (uint8_t*)cv.take((size_t)(L.cap + 1) * L.Cp) : nullptr;
      L.gmask = (L.kind == 2 && s >= 2 && Lb.kind == 1 && Lb.F == 2) ? (uint16_t*)cv.take((size_t)(L.cap + 1) * 2)
                                                                     : nullptr;
    } else {
      L.rules = L.rules_t = nullptr;
      L.argmax = nullptr;
      L.gmask = nullptr;
    }
    L.Xd = nullptr;
  }
  if (net->d.dropout)
    for (int s = 1; s < net->nlayers; ++s)
      if (net->L[s].drop_level >= 0) {
        LayerPlan& Lb = net->L[s - 1];
        Lb.Xd = cv.take((size_t)(Lb.cap + 1) * Lb.Cp * net->esz);
      }
  for (int p = 0; p < net->nparams; ++p) {
    ParamPlan& P = net->P[p];
    P.WpF = cv.take((size_t)P.NpadF * P.KpadF * net->esz);
    P.WpD = cv.take((size_t)P.NpadD * P.KpadD * net->esz);
    // every layer's partials coexist: the weight gradients run as one group
    P.part_off = max_part;
    if (P.nchunks > 1) max_part += (size_t)P.nchunks * P.Mpad_w * P.Npad_w;
    max_d0 = std::max(max_d0, (size_t)P.A * P.c_out);
    if (P.pf.ksplit > 1) max_gpart = std::max(max_gpart, (size_t)P.pf.ksplit * P.rows_f * P.pf.Npad);
    if (P.pd.ksplit > 1) max_gpart = std::max(max_gpart, (size_t)P.pd.ksplit * P.rows_d * P.pd.Npad);
  }
  const LayerPlan& Lt = net->L[net->nlayers - 1];
  net->dlogits = cv.take((size_t)B * net->dl_stride * net->esz);
  net->dh = (float*)cv.take((size_t)B * Lt.Cp * 4);
  net->loss_part = (float*)cv.take((size_t)B * 4);
  net->wpart = (float*)cv.take(std::max<size_t>(max_part, 1) * 4);
  net->gpart = (float*)cv.take(std::max<size_t>(max_gpart, 1) * 4);
  // two of each, by convolution parity: a launch may finish one convolution's
  // sums while it writes the next one's partials, or read the D0 of the
  // convolution above a pooling layer while it writes the one below
  net->d0_half = (max_d0 + 63) / 64 * 64;
  net->D0 = (float*)cv.take(2 * net->d0_half * 4);
  // (a pooling backward run in a GEMM epilogue keeps one partial per row tile:
  // up to 2 + 4 slots, cp channels, its row tiles at capacity)
  net->ppart_half = (size_t)net->pool_parts * (2 + 9) * max_cp;
  for (int s = 3; s < net->nlayers; ++s) {
    int bm = 0;
    const int64_t t = route_tiles(net, s, &bm);
    if (t > 0) net->ppart_half = std::max(net->ppart_half, (size_t)(2 + 4) * net->L[s - 2].Cp * (size_t)t);
  }
  net->ppart = (float*)cv.take(2 * net->ppart_half * 4);
  net->hdrop = net->d.dropout ? cv.take((size_t)B * Lt.Cp * net->esz) : nullptr;
  net->ws_bytes = cv.off + 256;
}

static void set_plan(GemmArgs& g, const GemmPlan& p, int64_t rows_cap, float* gpart) {
  g.cfg = p.cfg;
  g.sk = p.sk;
  g.ksplit = p.ksplit;
  g.part = gpart;
  g.part_rows = (int32_t)rows_cap;
}

// Most site chunks of a split-K weight gradient (the partial buffers hold that
// many): slabs x BK sites per chunk at the row capacity, at most 512, and
// partial sums (chunks x |dW| fp32) of at most twice the bytes the kernel reads
// (rows x row_bytes).  The kernel takes min(this, rows / (slabs x BK)) from the
// device-side row count.
static int wgrad_chunks(int64_t rows_cap, int slabs, int BK, int64_t row_bytes, int64_t part_bytes) {
  int64_t n = std::max<int64_t>(1, std::min<int64_t>(512, (rows_cap + slabs * BK - 1) / (slabs * BK)));
  return (int)std::min<int64_t>(n, std::max<int64_t>(1, 2 * rows_cap * row_bytes / std::max<int64_t>(part_bytes, 1)));
}

extern "C" {

const char* sscn_status_string(int32_t s) {
  switch (s) {
    case SSCN_OK: return "ok";
    case SSCN_ERR_INVALID_ARGUMENT: return "invalid argument";
    case SSCN_ERR_OUT_OF_RANGE: return "site outside the grid or batch";
    case SSCN_ERR_DUPLICATE_SITE: return "site listed twice";
    case SSCN_ERR_CAPACITY: return "batch or site count above the net's limits";
    case SSCN_ERR_BAD_STATE: return "call out of order";
    case SSCN_ERR_HIP: return "HIP runtime error";
    case SSCN_ERR_WORKSPACE: return "workspace null, too small or misaligned";
    default: return "unknown status";
  }
}

sscn_status sscn_net_create(const sscn_net_desc* desc, sscn_net** out) {
  if (!desc || !out) return SSCN_ERR_INVALID_ARGUMENT;
  *out = nullptr;
  const sscn_net_desc& d = *desc;
  if (d.ell < 1 || d.ell > 8 || d.k < 1 || d.c_in < 1 || d.n_classes < 1 || d.batch_max < 1 || d.max_active < 1)
    return SSCN_ERR_INVALID_ARGUMENT;
  if (d.dtype != SSCN_F32 && d.dtype != SSCN_BF16) return SSCN_ERR_INVALID_ARGUMENT;
  if (d.arch != SSCN_DEEPCNET && d.arch != SSCN_DEEPCNIN) return SSCN_ERR_INVALID_ARGUMENT;
  const int64_t N = 3ll << d.ell;
  if ((int64_t)d.batch_max * N * N >= (1ll << 31)) return SSCN_ERR_INVALID_ARGUMENT;
  if ((int64_t)(d.ell + 1) * d.k > (1 << 20) || d.n_classes > (1 << 24) || d.c_in > (1 << 16))
    return SSCN_ERR_INVALID_ARGUMENT;
  sscn_net* net = new (std::nothrow) sscn_net();
  if (!net) return SSCN_ERR_INVALID_ARGUMENT;
  net->d = d;
  net->bf16 = d.dtype == SSCN_BF16;
  net->esz = net->bf16 ? 2 : 4;
  net->VE = 16 / net->esz;
  const bool nin = d.arch == SSCN_DEEPCNIN;
  net->nin = nin;
  net->slope = nin ? 1.f / 3.f : 0.f;  // leaky rectifier x/3 (Section 2.2), else ReLU
  net->nlayers = nin ? 3 * d.ell + 3 : 2 * d.ell + 2;
  net->nconv = nin ? 2 * d.ell + 2 : d.ell + 1;
  net->nparams = net->nconv + 1;
  net->pool_parts = 1024;  // most row blocks per slot of a bias / ground-row reduction
  net->wgrad_slabs[0] = WG_SLABS_128;
  net->wgrad_slabs[1] = WG_SLABS_64;
  const int BK = net->bf16 ? 64 : 32;
  const int VE = net->VE;
  auto cp = [VE](int c) { return (int)round_up(c, VE); };
  // layers: input N; conv3 N-2; then (pool S/2, conv2 S-1) x ell (Section 2.1);
  // DeepCNiN adds a 1x1 convolution of the same width after every pool and after
  // the last convolution (Section 2.2)
  int kinds[MAX_LAYERS], Fs[MAX_LAYERS], widths[MAX_LAYERS];
  {
    int n = 0;
    kinds[n] = 1, Fs[n] = 3, widths[n] = d.k, ++n;
    for (int lv = 2; lv <= d.ell + 1; ++lv) {
      kinds[n] = 2, Fs[n] = 2, widths[n] = (lv - 1) * d.k, ++n;
      if (nin) kinds[n] = 1, Fs[n] = 1, widths[n] = (lv - 1) * d.k, ++n;
      kinds[n] = 1, Fs[n] = 2, widths[n] = lv * d.k, ++n;
    }
    if (nin) kinds[n] = 1, Fs[n] = 1, widths[n] = (d.ell + 1) * d.k, ++n;
    if (n + 1 != net->nlayers) {
      delete net;
      return SSCN_ERR_INVALID_ARGUMENT;
    }
  }
  LayerPlan* L = net->L;
  L[0] = LayerPlan{};
  L[0].kind = 0;
  L[0].S = (int)N;
  L[0].C = d.c_in;
  L[0].cap = d.max_active;
  int S = (int)N, C = d.c_in, ci = 0, dl = 0;
  L[0].drop_level = -1;
  for (int s = 1; s < net->nlayers; ++s) {
    LayerPlan& l = L[s];
    l = LayerPlan{};
    l.drop_level = (kinds[s - 1] == 1 && Fs[s - 1] > 1) ? dl++ : -1;
    const int64_t below = L[s - 1].cap;
    if (kinds[s - 1] == 1) {
      l.kind = 1;
      l.F = Fs[s - 1];
      l.S = S - (l.F - 1);
      l.C = widths[s - 1];
      l.conv_index = ci++;
    } else {
      // with N = 3 * 2^ell every pooling input side is even, so each site below
      // lies in exactly one window (the pooling backward relies on it)
      if (S % 2 != 0) {
        delete net;
        return SSCN_ERR_INVALID_ARGUMENT;
      }
      l.kind = 2;
      l.F = 2;
      l.S = S / 2;
      l.C = C;
      l.conv_index = -1;
    }
    l.A = l.F * l.F;
    const int64_t grid_cap = (int64_t)d.batch_max * l.S * l.S;
    l.cap = std::min<int64_t>(grid_cap, (l.kind == 1 ? l.A : 1) * below);
    S = l.S;
    C = l.C;
  }
  for (int s = 0; s < net->nlayers; ++s) {
    L[s].Cp = cp(L[s].C);
    if (L[s].Cp / VE > 256) {  // one channel vector per thread of a 256-thread block
      delete net;
      return SSCN_ERR_INVALID_ARGUMENT;
    }
    L[s].Wd = (L[s].S + 63) / 64;
    // 32-bit element offsets everywhere; bf16 feature rows and window lists
    // are also read through buffer descriptors whose byte range stops below 2^31
    const int64_t elems = (L[s].cap + 1) * (int64_t)std::max(L[s].Cp, std::max(L[s].A, 1));
    const int64_t rule_bytes = (L[s].cap + 1) * (int64_t)std::max(L[s].A, 1) * 4;  // window lists, read the same way
    if (elems >= (1ll << 31) || (net->bf16 && (elems * 2 > GATHER_SRC_BYTES || rule_bytes > GATHER_SRC_BYTES))) {
      delete net;
      return SSCN_ERR_INVALID_ARGUMENT;
    }
  }
  net->max_words = L[0].S * L[0].Wd;
  net->dl_stride = cp(d.n_classes);
  // parameters
  for (int s = 1; s < net->nlayers; ++s) {
    if (L[s].kind != 1) continue;
    ParamPlan& P = net->P[L[s].conv_index];
    P.A = L[s].A;
    P.c_in = L[s - 1].C;
    P.c_out = L[s].C;
    P.cp_in = L[s - 1].Cp;
    P.cp_out = L[s].Cp;
    P.rows_f = L[s].cap + 1;
    P.rows_d = L[s - 1].cap + 1;
    // a convolution under a pooling layer computes that layer in its epilogue
    const bool pooled = s + 1 < net->nlayers && L[s + 1].kind == 2;
    P.pf = plan_gemm(net->bf16, P.rows_f, P.c_out, P.A * P.cp_in, false, pooled ? 256 : 128);
    // an input gradient that is a pooling layer's may route its rows through the
    // pooling windows in its epilogue
    P.pd = plan_gemm(net->bf16, P.rows_d, P.c_in, P.A * P.cp_out, L[s - 1].kind == 2, 600);
    P.NpadF = P.pf.Npad;
    P.KpadF = P.pf.Kpad;
    P.NpadD = P.pd.Npad;
    P.KpadD = P.pd.Kpad;
    P.m_ones = -1;  // db comes from the bias / ground-row sums
    P.Mpad_w = (int)round_up(P.A * P.cp_in, WG_BM);
    P.bn_w = wgrad_bn(P.c_out);
    P.Npad_w = (int)round_up(P.c_out, P.bn_w);
    {
      const int m_rows = P.A * P.cp_in;
      const int64_t row_bytes = (int64_t)(P.A * P.cp_in + P.cp_out) * net->esz;
      const int64_t part_bytes = (int64_t)m_rows * P.Npad_w * 4;
      P.nchunks = wgrad_chunks(L[s].cap + 1, net->wgrad_slabs[P.bn_w == 128 ? 0 : 1], BK, row_bytes, part_bytes);
    }
  }
  {
    ParamPlan& P = net->P[net->nconv];
    const LayerPlan& Lt = L[net->nlayers - 1];
    P.A = 1;
    P.c_in = Lt.C;
    P.c_out = d.n_classes;
    P.cp_in = Lt.Cp;
    P.cp_out = net->dl_stride;
    P.rows_f = d.batch_max;
    P.rows_d = d.batch_max;
    P.pf = plan_gemm(net->bf16, P.rows_f, P.c_out, P.cp_in, false, 128);
    P.pd = plan_gemm(net->bf16, P.rows_d, P.c_in, P.cp_out, false, 128);
    P.NpadF = P.pf.Npad;
    P.KpadF = P.pf.Kpad;
    P.NpadD = P.pd.Npad;
    P.KpadD = P.pd.Kpad;
    P.m_ones = P.cp_in;
    P.Mpad_w = (int)round_up(P.m_ones + 1, WG_BM);
    P.bn_w = wgrad_bn(P.c_out);
    P.Npad_w = (int)round_up(P.c_out, P.bn_w);
    P.nchunks = 1;
  }
  if (dl != d.ell + 1) {
    delete net;
    return SSCN_ERR_INVALID_ARGUMENT;
  }
  carve(net, nullptr);
  *out = net;
  return SSCN_OK;
}

void sscn_net_destroy(sscn_net* net) { delete net; }

int32_t sscn_net_num_params(const sscn_net* net) { return net ? net->nparams : 0; }

sscn_status sscn_net_param_shape(const sscn_net* net, int32_t layer, int64_t* rows, int64_t* cols) {
  if (!net || !rows || !cols || layer < 0 || layer >= net->nparams) return SSCN_ERR_INVALID_ARGUMENT;
  const ParamPlan& P = net->P[layer];
  *rows = (int64_t)P.A * P.c_in;
  *cols = P.c_out;
  return SSCN_OK;
}

sscn_status sscn_net_workspace_bytes(const sscn_net* net, size_t* bytes) {
  if (!net || !bytes) return SSCN_ERR_INVALID_ARGUMENT;
  *bytes = net->ws_bytes;
  return SSCN_OK;
}

static sscn_status rulebook_build(sscn_net* net, const int32_t* d_coords, const int32_t* d_sample_begin, int32_t n,
                                  int32_t batch, void* d_ws, size_t ws_bytes, void* stream) {
  if (!net || n < 0 || batch < 0) return SSCN_ERR_INVALID_ARGUMENT;
  if (n > 0 && !d_coords) return SSCN_ERR_INVALID_ARGUMENT;
  if (n > net->d.max_active || batch > net->d.batch_max) return SSCN_ERR_CAPACITY;
  if (!d_ws || ws_bytes < net->ws_bytes || ((uintptr_t)d_ws & 255u)) return SSCN_ERR_WORKSPACE;
  net->built = net->forwarded = net->backwarded = false;
  hipStream_t st = (hipStream_t)stream;
  if (net->ws != d_ws) {
    carve(net, d_ws);
    net->ws = d_ws;
    net->rb_parity = 0;
    const LayerPlan& L0 = net->L[0];
    if (launch_rulebook_reset(L0.bits, net->bits0_alt, (int64_t)net->d.batch_max * L0.S * L0.Wd, net->err, st) !=
        hipSuccess)
      return SSCN_ERR_HIP;
  }
  net->batch = batch;
  net->n = n;
  RulebookArgs a;
  std::memset(&a, 0, sizeof(a));
  a.nlayers = net->nlayers;
  a.batch = batch;
  for (int s = 0; s < net->nlayers; ++s) {
    const LayerPlan& L = net->L[s];
    a.L[s] = LayerBits{L.bits, L.wpre, L.scount, L.soff, L.sites, L.S, L.Wd};
    a.kind[s] = L.kind;
    a.F[s] = L.F;
    a.rules[s] = L.rules;
    a.rules_t[s] = L.rules_t;
    a.gmask[s] = L.gmask;
  }
  // composite windows: a valid F x F convolution widens the square by F - 1
  // steps of the layer below, a 2 x 2 stride-2 pooling by one step and doubles
  // the step
  a.rf_a[0] = 1, a.rf_r[0] = 1;
  for (int s = 1; s < net->nlayers; ++s) {
    const LayerPlan& L = net->L[s];
    a.rf_a[s] = L.kind == 2 ? 2 * a.rf_a[s - 1] : a.rf_a[s - 1];
    a.rf_r[s] = a.rf_r[s - 1] + a.rf_a[s - 1] * (L.F - 1);
  }
  a.counts = net->counts;
  // this build's input bitmap and error word, and the next build's (cleared
  // here); err[1] is the loss counter, err[0] the label-error word of the
  // training forward passes (cleared by the sscn_layer_sizes that reports it)
  const int par = net->rb_parity;
  uint64_t* bits0[2] = {net->L[0].bits, net->bits0_alt};
  a.L[0].bits = bits0[par];
  a.bits0_next = bits0[1 - par];
  a.err = net->err + 2 + par;
  a.err_next = net->err + 2 + (1 - par);
  a.batch_max = net->d.batch_max;
  net->err_cur = a.err;
  a.perm = net->perm;
  a.head_rows = net->head_rows;
  a.coords = d_coords;
  a.n = n;
  a.sample_begin = batch > 0 ? d_sample_begin : nullptr;
  // window-list segments: LISTS_WPB bitmap words of a layer per workgroup (one
  // workgroup for an empty batch, which writes the ground rows), 256 caller
  // sites or samples per workgroup
  ListsWork lw;
  std::memset(&lw, 0, sizeof(lw));
  auto add_seg = [&](int kind, int layer, int64_t blocks) {
    lw.kind[lw.nseg] = kind;
    lw.layer[lw.nseg] = layer;
    lw.blk[lw.nseg + 1] = lw.blk[lw.nseg] + (int)std::max<int64_t>(1, blocks);
    ++lw.nseg;
  };
  for (int s = 0; s < net->nlayers; ++s)
    add_seg(0, s, ((int64_t)batch * net->L[s].S * net->L[s].Wd + LISTS_WPB - 1) / LISTS_WPB);
  add_seg(2, 0, ((int64_t)n + 255) / 256);
  add_seg(3, 0, ((int64_t)batch + 255) / 256);
  if (timed(net, SSCN_KC_RULEBOOK, st, [&] { return launch_rulebook(a, lw, net->max_words, st); }) != hipSuccess)
    return SSCN_ERR_HIP;
  net->rb_parity = 1 - par;
  net->built = true;
  return SSCN_OK;
}

sscn_status sscn_rulebook_build(sscn_net* net, const int32_t* d_coords, int32_t n, int32_t batch, void* d_ws,
                                size_t ws_bytes, void* stream) {
  return rulebook_build(net, d_coords, nullptr, n, batch, d_ws, ws_bytes, stream);
}

sscn_status sscn_rulebook_build_grouped(sscn_net* net, const int32_t* d_coords, const int32_t* d_sample_begin, int32_t n,
                                        int32_t batch, void* d_ws, size_t ws_bytes, void* stream) {
  if (!d_sample_begin) return SSCN_ERR_INVALID_ARGUMENT;
  return rulebook_build(net, d_coords, d_sample_begin, n, batch, d_ws, ws_bytes, stream);
}

sscn_status sscn_layer_sizes(sscn_net* net, int32_t* h_counts, void* stream) {
  if (!net || !h_counts) return SSCN_ERR_INVALID_ARGUMENT;
  if (!net->built) return SSCN_ERR_BAD_STATE;
  hipStream_t st = (hipStream_t)stream;
  int32_t err = 0, label_err = 0;
  if (hipMemcpyAsync(h_counts, net->counts, sizeof(int32_t) * net->nlayers, hipMemcpyDeviceToHost, st) != hipSuccess)
    return SSCN_ERR_HIP;
  if (hipMemcpyAsync(&err, net->err_cur, sizeof(int32_t), hipMemcpyDeviceToHost, st) != hipSuccess) return SSCN_ERR_HIP;
  if (hipMemcpyAsync(&label_err, net->err, sizeof(int32_t), hipMemcpyDeviceToHost, st) != hipSuccess)
    return SSCN_ERR_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return SSCN_ERR_HIP;
  if (label_err) {  // an earlier training forward saw a label outside [0, n_classes): report it once
    static const int32_t zero = 0;
    if (hipMemcpyAsync(net->err, &zero, sizeof(int32_t), hipMemcpyHostToDevice, st) != hipSuccess ||
        hipStreamSynchronize(st) != hipSuccess)
      return SSCN_ERR_HIP;
    return SSCN_ERR_OUT_OF_RANGE;
  }
  if (err & ERRBIT_RANGE) return SSCN_ERR_OUT_OF_RANGE;
  if (err & ERRBIT_DUP) return SSCN_ERR_DUPLICATE_SITE;
  return SSCN_OK;
}

// Dropout of level j in the current pass (off unless a training pass with rate > 0).
static DropArgs drop_args(const sscn_net* net, int j, const int32_t* keys) {
  DropArgs d{};
  if (!net->drop_on || j < 0 || j >= net->n_rates || !(net->rates[j] > 0.0)) return d;
  const double p = net->rates[j];
  d.keys = keys;
  d.thr = (uint32_t)std::floor(p * 4294967296.0);
  d.level = (uint32_t)j;
  d.seed_lo = (uint32_t)net->seed;
  d.seed_hi = (uint32_t)(net->seed >> 32);
  d.scale = (float)(1.0 / (1.0 - p));
  d.on = 1;
  return d;
}

// Dropout on the input of convolution s (rows of layer s - 1, keyed by its sites).
static DropArgs conv_drop(const sscn_net* net, int s) {
  return drop_args(net, net->L[s].drop_level, net->L[s - 1].sites);
}

// Dropout on the softmax layer's input (the last level, keyed by sample).
static DropArgs head_drop(const sscn_net* net) { return drop_args(net, net->d.ell + 1, nullptr); }

// Whether convolution s runs the pooling layer above it in its GEMM epilogue
// (GemmArgs::pool_fwd): every site of the convolution must lie in a pooling
// window (an even grid side), and its plan must be a single-pass tile shape
// that stages its output.
static bool pool_fused(const sscn_net* net, int s) {
  if (s + 1 >= net->nlayers) return false;
  const LayerPlan& L = net->L[s];
  const LayerPlan& Lp = net->L[s + 1];
  if (L.kind != 1 || Lp.kind != 2 || L.S % 2 != 0 || Lp.Cp != L.Cp) return false;
  const ParamPlan& P = net->P[L.conv_index];
  return P.pf.ksplit == 1 && gemm_routes(net->bf16, P.pf.cfg);
}

// Stage s of the forward pass; with fuse_pool a convolution whose pooling
// layer above pool_fused allows also computes that layer (whose own stage is
// then skipped).
static hipError_t forward_stage(sscn_net* net, int s, hipStream_t st, bool fuse_pool = false) {
  const LayerPlan& L = net->L[s];
  const LayerPlan& Lb = net->L[s - 1];
  if (L.kind == 1) {
    const ParamPlan& P = net->P[L.conv_index];
    const DropArgs dr = conv_drop(net, s);
    if (dr.on) {
      const hipError_t e = timed(net, SSCN_KC_DROPOUT, st, [&] {
        return launch_dropout_rows(net->bf16, Lb.X, Lb.Xd, Lb.Cp, net->counts + s - 1, Lb.cap + 1, dr, st);
      });
      if (e != hipSuccess) return e;
    }
    GemmArgs g{};
    g.src = dr.on ? Lb.Xd : Lb.X;
    g.src_stride = Lb.Cp;
    g.rmap = L.rules;
    g.A = L.A;
    g.cseg = Lb.Cp;
    g.K = L.A * Lb.Cp;
    g.Kpad = P.KpadF;
    g.Bt = P.WpF;
    g.Npad = P.NpadF;
    g.bias = net->b[L.conv_index];
    g.N = L.C;
    g.out_cols = L.Cp;
    g.out = L.X;
    g.out_stride = L.Cp;
    g.epi = net->slope == 0.f ? EPI_BIAS_RELU : EPI_BIAS_LRELU;
    if (L.A == 1) g.rmap = nullptr;  // a 1x1 layer reads its own row of the layer below
    g.rows_dev = net->counts + s;
    g.rows_add = 1;
    g.row_begin = 0;
    set_plan(g, P.pf, P.rows_f, net->gpart);
    int64_t max_rows = L.cap + 1;
    if (fuse_pool && pool_fused(net, s)) {  // rows: the four slots of every pooling window
      const LayerPlan& Lp = net->L[s + 1];
      g.pool_fwd = 1;
      g.pslot = Lp.rules;
      g.pool_out = Lp.X;
      g.pool_argmax = Lp.argmax;
      g.pool_stride = Lp.Cp;
      g.rows_dev = net->counts + s + 1;
      max_rows = 4 * (Lp.cap + 1);
    }
    if (conv_narrow_ok(net->bf16, g, Lb.C))  // few input channels: no GEMM
      return timed(
          net, SSCN_KC_CONV_NARROW, st, [&] { return launch_conv_narrow(net->bf16, g, Lb.C, max_rows, st); },
          launch_tag(s, SSCN_ROLE_FORWARD, SSCN_PLAN_NONE, false, g.pool_fwd != 0));
    return timed_gemm(net, g, max_rows, st, s, SSCN_ROLE_FORWARD);
  }
  return timed(net, SSCN_KC_POOL_FWD, st, [&] {
    return launch_pool_fwd(net->bf16, Lb.X, Lb.Cp, L.rules, L.X, L.Cp, L.argmax, L.Cp, net->counts + s, L.cap, st);
  });
}

// Row blocks of a bias / ground-row reduction over `rows` rows: about 8 rows
// per thread.
static int ground_parts(const sscn_net* net, int64_t rows, int cp) {
  const int lanes = 256 / (cp / (net->bf16 ? 8 : 4));
  return (int)std::min<int64_t>(net->pool_parts, std::max<int64_t>(1, (rows + 8 * lanes - 1) / (8 * lanes)));
}

// Blocks of the fused pooling backward over `rows` pooling rows: one row per
// thread and at most 512 blocks (more rows per thread beyond that).
static int pool_bwd_blocks(const sscn_net* net, int64_t rows, int cp) {
  const int lanes = 256 / (cp / (net->bf16 ? 8 : 4));
  return (int)std::min<int64_t>(std::min(512, net->pool_parts), std::max<int64_t>(1, (rows + lanes - 1) / lanes));
}

// Slot partials and ground sums D0 of convolution s (alternating halves).
static float* part_of(const sscn_net* net, int s) {
  return net->ppart + (size_t)(net->L[s].conv_index & 1) * net->ppart_half;
}
static float* d0_of(const sscn_net* net, int s) {
  return net->D0 + (size_t)(net->L[s].conv_index & 1) * net->d0_half;
}

// Whether the backward pass needs row 0 of the gradient below convolution s
// (the ground row of its input): always above the first layer; for the first,
// only when the caller asks for the input-feature gradient, which its
// layer view then holds in full.
static bool needs_row0(const sscn_net* net, int s) { return s > 1 || net->want_dfeats; }

// Bias / ground-row reduction arguments of convolution s (pool_above: pooling
// layer s+1 sits on it and routes its gradient; its windows give slot 0).
static GroundArgs ground_args(const sscn_net* net, int s, bool pool_above) {
  const LayerPlan& L = net->L[s];
  const int ci = L.conv_index;
  GroundArgs g{};
  if (pool_above) {
    const LayerPlan& Lp = net->L[s + 1];
    g.dY = Lp.grad;
    g.argmax = Lp.argmax;
    g.Rp = Lp.rules;
    g.n_pool = net->counts + s + 1;
    g.B1 = pool_bwd_blocks(net, Lp.cap, Lp.Cp);
    g.B2 = g.B1;  // one pass: the fused pooling backward
    g.Y_below = L.X;
    g.X_pool = Lp.X;
    g.gmask = Lp.gmask;
  } else {
    g.B2 = ground_parts(net, L.cap, L.Cp);
  }
  g.dZ = L.grad;
  g.R = L.rules;
  g.n_rows = net->counts + s;
  g.stride = L.Cp;
  g.cp = L.Cp;
  g.c_out = L.C;
  g.part = part_of(net, s);
  g.PM = net->pool_parts;
  g.slope = net->slope;
  g.db = net->db[ci];
  g.D0 = d0_of(net, s);
  return g;
}

// Row 0 of convolution s's output gradient delta (with a pooling layer above:
// its fused backward has written the partial sums), the bias gradient and the
// ground-row sums, then row 0 of the gradient below.
static hipError_t ground_level(sscn_net* net, int s, bool pool_above, hipStream_t st) {
  const LayerPlan& L = net->L[s];
  const LayerPlan& Lb = net->L[s - 1];
  const int ci = L.conv_index;
  const ParamPlan& P = net->P[ci];
  // a 1x1 layer's input-gradient GEMM covers row 0 itself (its window is the row)
  const bool row0 = needs_row0(net, s) && L.A > 1;
  const GroundArgs g = ground_args(net, s, pool_above);
  hipError_t e;
  if ((e = timed(net, SSCN_KC_GROUND, st, [&] {
         return launch_ground(net->bf16, g, row0 ? L.A : 0, pool_above ? 2 : 0, st);
       })) != hipSuccess)
    return e;
  if (!row0) return hipSuccess;
  // below a convolution the stored gradient is dL/dZ: times its rectifier derivative
  const void* mask = Lb.kind == 1 ? Lb.X : nullptr;
  return timed(net, SSCN_KC_GROUND, st, [&] {
    return launch_row0_dx(net->bf16, net->W[ci], d0_of(net, s), P.A, P.c_in, P.c_out, Lb.Cp, Lb.grad, mask, net->slope,
                          st);
  });
}

// The final ground pass of convolution s as an extra task.
static ExtraTask final_task(const sscn_net* net, int s, bool pool_above) {
  const LayerPlan& L = net->L[s];
  ExtraTask x{};
  x.kind = 1;
  x.blocks = L.Cp;
  x.AC = (needs_row0(net, s) && L.A > 1) ? L.A : 0;
  x.g = ground_args(net, s, pool_above);
  return x;
}

// Row 0 of the gradient below convolution s as an extra task (reads D0 from
// its final pass, which must have run in an earlier launch).
static ExtraTask row0_task(const sscn_net* net, int s) {
  const LayerPlan& L = net->L[s];
  const LayerPlan& Lb = net->L[s - 1];
  const ParamPlan& P = net->P[L.conv_index];
  ExtraTask x{};
  x.kind = 2;
  x.blocks = Lb.Cp;
  x.r = Row0Args{net->W[L.conv_index], d0_of(net, s), P.A, P.c_in, P.c_out, Lb.Cp, Lb.grad,
                 Lb.kind == 1 ? Lb.X : nullptr, net->slope};
  return x;
}

// Weight-gradient arguments of convolution s (run once its delta is complete).
static WGradArgs conv_wgrad_args(const sscn_net* net, int s) {
  const LayerPlan& L = net->L[s];
  const LayerPlan& Lb = net->L[s - 1];
  const int ci = L.conv_index;
  const ParamPlan& P = net->P[ci];
  WGradArgs w{};
  w.src = conv_drop(net, s).on ? Lb.Xd : Lb.X;  // the input the forward pass used
  w.src_stride = Lb.Cp;
  w.rmap = L.rules;
  w.A = L.A;
  w.cseg = Lb.Cp;
  w.m_ones = P.m_ones;
  w.Mpad = P.Mpad_w;
  w.dsrc = L.grad;
  w.dsrc_stride = L.Cp;
  w.dsrc_cols = L.Cp;
  w.Npad = P.Npad_w;
  w.rows_dev = net->counts + s;
  w.rows_add = 1;
  w.nchunks = P.nchunks;
  w.slabs = net->wgrad_slabs[P.bn_w == 128 ? 0 : 1];
  w.part = net->wpart + P.part_off;
  w.cfg = P.bn_w == 128 ? 0 : 1;
  w.dW = net->dW[ci];
  w.db = net->db[ci];
  w.c_in = P.c_in;
  w.c_out = P.c_out;
  return w;
}

// Weight gradients of a list of layers: one launch per tile shape, then one
// launch reducing every split-K layer.  A ground final pass that must precede
// layer fin_layer's weight gradient (it writes that layer's delta row 0) rides
// on the first launch when that launch does not hold fin_layer, else runs alone
// first.
static hipError_t run_wgrads(sscn_net* net, const WGradArgs* w, int n, hipStream_t st,
                             const ExtraTask* fin = nullptr, int fin_layer = -1) {
  hipError_t e;
  bool fin_done = !fin || !fin->kind;
  for (int cfg = 0; cfg < 2; ++cfg) {
    WGradArgs sel[MAX_WG_LAYERS];
    int k = 0;
    bool holds = false;
    for (int i = 0; i < n; ++i)
      if (w[i].cfg == cfg) {
        holds = holds || i == fin_layer;
        sel[k++] = w[i];
      }
    if (!k) continue;
    const ExtraTask* x = nullptr;
    if (!fin_done) {
      if (holds) {
        if ((e = timed(net, SSCN_KC_GROUND, st, [&] { return launch_extra(net->bf16, *fin, st); })) != hipSuccess)
          return e;
      } else {
        x = fin;
      }
      fin_done = true;
    }
    if ((e = timed(net, SSCN_KC_WGRAD, st, [&] { return launch_wgrad(net->bf16, cfg, sel, k, st, x); })) !=
        hipSuccess)
      return e;
  }
  if (!fin_done &&
      (e = timed(net, SSCN_KC_GROUND, st, [&] { return launch_extra(net->bf16, *fin, st); })) != hipSuccess)
    return e;
  return timed(net, SSCN_KC_WGRAD_REDUCE, st, [&] { return launch_wgrad_reduce(net->bf16, w, n, st); });
}

// Whether the input-gradient GEMM of convolution s, when it computes the
// gradient of a pooling layer s-1 on convolution s-2, runs that pooling
// layer's backward in its epilogue (GemmArgs::route): not through a dropout of
// the pooling output, not for a 3x3 convolution below that must finish its
// nine ground sums, and only for a tile shape that stages its output with one
// partial per row tile (*bm rows, *tiles at capacity).
static bool route_into(const sscn_net* net, int s, int* ac, int* bm, int* tiles) {
  int b = 0;
  const int64_t t = route_tiles(net, s, &b);
  if (t < 1 || !needs_row0(net, s) || conv_drop(net, s).on) return false;
  const LayerPlan& Lc = net->L[s - 2];
  const int a = (needs_row0(net, s - 2) && Lc.A > 1) ? Lc.A : 0;
  if (a != 0 && a != 4) return false;
  if ((size_t)(2 + a) * Lc.Cp * (size_t)t > net->ppart_half || t > (1 << 30)) return false;
  *ac = a;
  *bm = b;
  *tiles = (int)t;
  return true;
}

// Rows >= 1 of the gradient below stage s: the pooling backward (with the
// partial sums of the convolution below), or the input-gradient GEMM of a
// convolution.  (The GEMM reads delta rows >= 1 only: a window list entry of -1
// selects zero, whatever its load of row 0 returned.)  With allow_route the
// GEMM also runs the pooling backward below it where route_into allows, and
// *routed says whether it did.
static hipError_t rows_below(sscn_net* net, int s, hipStream_t st, const ExtraTask* extra = nullptr,
                             bool allow_route = false, bool* routed = nullptr) {
  if (routed) *routed = false;
  const LayerPlan& L = net->L[s];
  const LayerPlan& Lb = net->L[s - 1];
  if (L.kind == 2) {
    // rows >= 1 below with the partial sums of the convolution below
    if (Lb.kind != 1) return hipErrorInvalidValue;  // a pooling layer sits on a convolution
    const GroundArgs g = ground_args(net, s - 1, true);
    const int Ac = (needs_row0(net, s - 1) && Lb.A > 1) ? Lb.A : 0;
    return timed(net, SSCN_KC_POOL_BWD, st, [&] { return launch_ground(net->bf16, g, Ac, 1, st, extra); });
  }
  if (!(s > 1 || net->want_dfeats)) return hipSuccess;
  const ParamPlan& P = net->P[L.conv_index];
  GemmArgs g{};
  g.src = L.grad;
  g.src_stride = L.Cp;
  g.rmap = L.rules_t;
  g.A = L.A;
  g.cseg = L.Cp;
  g.K = L.A * L.Cp;
  g.Kpad = P.KpadD;
  g.Bt = P.WpD;
  g.Npad = P.NpadD;
  g.bias = nullptr;
  g.N = Lb.C;
  g.out_cols = Lb.Cp;
  g.out = Lb.grad;
  g.out_stride = Lb.Cp;
  g.epi = EPI_STORE;
  if (Lb.kind == 1) {  // a convolution below: store dL/dZ, the rectifier derivative applied
    g.epi = EPI_STORE_MASK;
    g.mask = Lb.X;
    g.mask_stride = Lb.Cp;
    g.slope = net->slope;
  }
  if (extra) g.x = *extra;
  g.rows_dev = net->counts + s - 1;
  g.rows_add = 1;
  g.row_begin = 1;
  if (L.A == 1) {  // 1x1 layer: row i below takes row i's gradient, ground row included
    g.rmap = nullptr;
    g.row_begin = 0;
  }
  set_plan(g, P.pd, P.rows_d, net->gpart);
  int rac = 0, rbm = 0, rtiles = 0;
  if (allow_route && route_into(net, s, &rac, &rbm, &rtiles)) {
    g.route = 1;
    g.route_ac = rac;
    g.pr = ground_args(net, s - 2, true);
    g.pr.PM = rtiles;  // one partial per row tile
    if (routed) *routed = true;
  }
  hipError_t e = timed_gemm(net, g, Lb.cap + 1, st, s, SSCN_ROLE_INPUT_GRAD);
  const DropArgs dr = conv_drop(net, s);
  if (e == hipSuccess && dr.on)  // through the dropout of this convolution's input: rows >= 1, in place
    e = timed(net, SSCN_KC_DROPOUT, st, [&] {
      return launch_dropout_rows(net->bf16, Lb.grad, Lb.grad, Lb.Cp, net->counts + s - 1, Lb.cap + 1, dr, st);
    });
  return e;
}

sscn_status sscn_forward(sscn_net* net, const void* d_feats, const void* const* h_W, const float* const* h_b,
                         const int32_t* d_labels, float* d_logits, float* d_loss, void* stream) {
  if (!net || !h_W || !h_b || !d_logits) return SSCN_ERR_INVALID_ARGUMENT;
  if ((d_labels == nullptr) != (d_loss == nullptr)) return SSCN_ERR_INVALID_ARGUMENT;
  const bool train = d_labels != nullptr;  // else inference: logits only
  if (net->n > 0 && !d_feats) return SSCN_ERR_INVALID_ARGUMENT;
  if (!net->built) return SSCN_ERR_BAD_STATE;
  for (int p = 0; p < net->nparams; ++p)
    if (!h_W[p] || !h_b[p]) return SSCN_ERR_INVALID_ARGUMENT;
  hipStream_t st = (hipStream_t)stream;
  for (int p = 0; p < net->nparams; ++p) {
    net->W[p] = h_W[p];
    net->b[p] = h_b[p];
  }
  net->logits = d_logits;
  net->labels = d_labels;
  net->drop_on = train && net->n_rates > 0;
  net->backwarded = false;
  const LayerPlan& L0 = net->L[0];
  // the weight packings, with the input scatter as extra workgroups of the launch
  PackArgs pa;
  std::memset(&pa, 0, sizeof(pa));
  pa.sc = ScatterArgs{d_feats, net->n, net->d.c_in, net->perm, L0.X, L0.Cp, 0};
  for (int p = net->nparams - 1; p >= 0; --p) {  // the largest (softmax layer) first: its tiles find their job at once
    const ParamPlan& P = net->P[p];
    pa.job[pa.njobs++] = PackJob{h_W[p], P.WpF, 0, P.A, P.c_in, P.c_out, P.cp_in, P.cp_out, P.NpadF, P.KpadF};
    if (train)  // the input-gradient layout is only read by the backward pass
      pa.job[pa.njobs++] = PackJob{h_W[p], P.WpD, 1, P.A, P.c_in, P.c_out, P.cp_in, P.cp_out, P.NpadD, P.KpadD};
  }
  if (timed(net, SSCN_KC_HEAD, st, [&] { return launch_pack_all(net->bf16, pa, st); }) != hipSuccess)
    return SSCN_ERR_HIP;
  for (int s = 1; s < net->nlayers; ++s) {
    if (net->L[s].kind == 2 && pool_fused(net, s - 1)) continue;  // computed by the convolution below
    if (forward_stage(net, s, st, true) != hipSuccess) return SSCN_ERR_HIP;
  }
  // softmax layer on each sample's top-layer row
  const LayerPlan& Lt = net->L[net->nlayers - 1];
  const ParamPlan& P = net->P[net->nconv];
  const DropArgs hdr = head_drop(net);
  if (hdr.on && timed(net, SSCN_KC_DROPOUT, st, [&] {
        return launch_head_drop(net->bf16, Lt.X, net->head_rows, net->batch, Lt.Cp, net->hdrop, hdr, st);
      }) != hipSuccess)
    return SSCN_ERR_HIP;
  GemmArgs g{};
  g.src = hdr.on ? net->hdrop : Lt.X;
  g.src_stride = Lt.Cp;
  g.rmap = hdr.on ? nullptr : net->head_rows;
  g.A = 1;
  g.cseg = Lt.Cp;
  g.K = Lt.Cp;
  g.Kpad = P.KpadF;
  g.Bt = P.WpF;
  g.Npad = P.NpadF;
  g.bias = h_b[net->nconv];
  g.N = net->d.n_classes;
  g.out_cols = net->d.n_classes;
  g.out = d_logits;
  g.out_stride = net->d.n_classes;
  g.epi = EPI_BIAS_F32;
  g.rows_host = net->batch;
  g.row_begin = 0;
  set_plan(g, P.pf, P.rows_f, net->gpart);
  net->forwarded = false;
  if (timed_gemm(net, g, net->batch, st, 0, SSCN_ROLE_SOFTMAX_FWD) != hipSuccess)
    return SSCN_ERR_HIP;
  if (!train) return SSCN_OK;
  if (timed(net, SSCN_KC_HEAD, st, [&] {
        return launch_softmax_xent(net->bf16, d_logits, d_labels, net->batch, net->d.n_classes, net->dlogits,
                                   net->dl_stride, net->loss_part, d_loss, net->err + 1, net->err, st);
      }) != hipSuccess)
    return SSCN_ERR_HIP;
  net->forwarded = true;
  return SSCN_OK;
}

sscn_status sscn_backward(sscn_net* net, float* const* h_dW, float* const* h_db, void* d_dfeats, void* stream) {
  if (!net || !h_dW || !h_db) return SSCN_ERR_INVALID_ARGUMENT;
  if (!net->forwarded) return SSCN_ERR_BAD_STATE;
  for (int p = 0; p < net->nparams; ++p) {
    if (!h_dW[p] || !h_db[p]) return SSCN_ERR_INVALID_ARGUMENT;
    net->dW[p] = h_dW[p];
    net->db[p] = h_db[p];
  }
  hipStream_t st = (hipStream_t)stream;
  net->want_dfeats = d_dfeats != nullptr;
  const int top = net->nlayers - 1;
  const LayerPlan& Lt = net->L[top];
  const int fc = net->nconv;
  const ParamPlan& P = net->P[fc];
  // softmax layer: dh = dlogits W^T, scattered to the top layer's rows
  GemmArgs g{};
  g.src = net->dlogits;
  g.src_stride = net->dl_stride;
  g.rmap = nullptr;
  g.A = 1;
  g.cseg = net->dl_stride;
  g.K = net->dl_stride;
  g.Kpad = P.KpadD;
  g.Bt = P.WpD;
  g.Npad = P.NpadD;
  g.bias = nullptr;
  g.N = Lt.C;
  g.out_cols = Lt.Cp;
  g.out = net->dh;
  g.out_stride = Lt.Cp;
  g.epi = EPI_F32;
  g.rows_host = net->batch;
  g.row_begin = 0;
  set_plan(g, P.pd, P.rows_d, net->gpart);
  g.partials_only = g.ksplit > 1;  // the head backward sums the split-K partials itself
  if (timed_gemm(net, g, net->batch, st, 0, SSCN_ROLE_SOFTMAX_DH) != hipSuccess)
    return SSCN_ERR_HIP;
  // the head backward (scatter of dh into the top layer, with its ground sums)
  // runs in the stage loop below as the top convolution's sums launch
  HeadBwdArgs hb{};
  hb.dh_part = g.ksplit > 1 ? net->gpart : net->dh;
  hb.ksplit = g.ksplit;
  hb.ks_stride = (int64_t)g.part_rows * g.Npad;
  hb.dh_stride = g.ksplit > 1 ? g.Npad : Lt.Cp;
  hb.head_rows = net->head_rows;
  hb.batch = net->batch;
  hb.Y_top = Lt.X;
  hb.grad_top = Lt.grad;
  hb.cp = Lt.Cp;
  hb.slope = net->slope;
  hb.drop = head_drop(net);
  hb.R = Lt.rules;
  hb.part = part_of(net, top);
  hb.PM = net->pool_parts;
  // Stages from the top down, all on the caller's stream.  Per convolution:
  // its bias and ground-row sums (with a pooling layer above they come out of
  // that layer's backward), rows >= 1 of the gradient below, the final ground
  // pass (row 0 of delta, db, D0) and row 0 of the gradient below.  The final
  // pass needs only the sums and rides as extra workgroups on the input-gradient
  // GEMM, which reads delta rows >= 1 only (a 1x1 layer's GEMM reads row 0 too:
  // it rides there only when the pass does not rewrite row 0); row 0 below needs
  // D0 and rides on the next launch.
  //
  // A pooling layer's backward runs in the epilogue of the GEMM that computes
  // its gradient where route_into allows: its row 0 (row 0 below the
  // convolution above) then cannot ride on the next launch, whose final pass
  // reads it, and is computed by that final pass itself (extra task kind 3).
  ExtraTask pending{};  // row 0 of a gradient below, waiting for the next launch
  ExtraTask pool_row0{};  // row 0 of a routed pooling layer's gradient, for the final pass below it
  ExtraTask deferred_fin{};  // the first layer's final pass, when no launch of the stage loop follows it
  bool routed[MAX_LAYERS] = {};
  for (int s = top; s >= 1; --s) {
    const LayerPlan& L = net->L[s];
    hipError_t e = hipSuccess;
    if (L.kind == 2) {
      if (routed[s]) {
        pool_row0 = pending;
        pending = ExtraTask{};
        if (pool_row0.kind != 2) return SSCN_ERR_HIP;
        continue;
      }
      e = rows_below(net, s, st, pending.kind ? &pending : nullptr);
      pending = ExtraTask{};
    } else {
      const bool pool_above = s < top && net->L[s + 1].kind == 2;
      const bool row0 = needs_row0(net, s) && L.A > 1;
      ExtraTask fin = final_task(net, s, pool_above);
      if (pool_above && routed[s + 1]) {  // partials from the routed GEMM above, its row 0 computed here
        int rac = 0, rbm = 0, rtiles = 0;
        if (!route_into(net, s + 2, &rac, &rbm, &rtiles) || pool_row0.kind != 2) return SSCN_ERR_HIP;
        fin.g.B1 = fin.g.B2 = fin.g.PM = rtiles;
        fin.g.route_bm = rbm;
        fin.kind = 3;
        fin.r = pool_row0.r;
        pool_row0 = ExtraTask{};
      }
      if (s == top) {  // the head backward writes delta and its sums
        fin.g.B1 = fin.g.B2 = head_backward_parts(net->batch);
        fin.g.dY = L.grad;  // row 0 zeroed by the head backward
        fin.g.Y_below = L.X;
        if (pending.kind) return SSCN_ERR_HIP;  // nothing precedes the top layer
        e = timed(net, SSCN_KC_HEAD, st, [&] { return launch_head_backward(net->bf16, hb, fin.AC, st); });
      } else if (!pool_above) {  // the sums over delta rows, as their own launch
        const GroundArgs g = ground_args(net, s, false);
        e = timed(net, SSCN_KC_GROUND, st, [&] {
          return launch_ground(net->bf16, g, fin.AC, 3, st, pending.kind ? &pending : nullptr);
        });
        pending = ExtraTask{};
      }
      const bool gemm_below = s > 1 || net->want_dfeats;
      // the final pass writes row 0 of delta when it finishes a pooling layer's (or
      // the head's) sums: then only a GEMM that does not read row 0 may carry it
      const bool writes_row0 = pool_above || s == top;
      if (e == hipSuccess && gemm_below && (L.A > 1 || !writes_row0)) {
        e = rows_below(net, s, st, &fin, true, s >= 2 ? &routed[s - 1] : nullptr);
      } else if (e == hipSuccess && !gemm_below && s == 1) {
        // the first layer's final pass: on the weight-gradient launches at the end
        if (pending.kind) e = timed(net, SSCN_KC_GROUND, st, [&] { return launch_extra(net->bf16, pending, st); });
        pending = ExtraTask{};
        deferred_fin = fin;
      } else if (e == hipSuccess) {
        if (fin.kind == 3) {  // the final pass with its row 0 above, as a launch of its own
          if (pending.kind)
            e = timed(net, SSCN_KC_GROUND, st, [&] { return launch_extra(net->bf16, pending, st); });
          if (e == hipSuccess) e = timed(net, SSCN_KC_GROUND, st, [&] { return launch_extra(net->bf16, fin, st); });
        } else {
          const GroundArgs g = fin.g;
          e = timed(net, SSCN_KC_GROUND, st, [&] {
            return launch_ground(net->bf16, g, fin.AC, 2, st, pending.kind ? &pending : nullptr);
          });
        }
        pending = ExtraTask{};
        if (e == hipSuccess && gemm_below) e = rows_below(net, s, st, nullptr, true, s >= 2 ? &routed[s - 1] : nullptr);
      }
      if (row0) pending = row0_task(net, s);
    }
    if (e != hipSuccess) return SSCN_ERR_HIP;
  }
  if (pending.kind &&
      timed(net, SSCN_KC_GROUND, st, [&] { return launch_extra(net->bf16, pending, st); }) != hipSuccess)
    return SSCN_ERR_HIP;
  if (d_dfeats) {
    const LayerPlan& L0 = net->L[0];
    if (timed(net, SSCN_KC_HEAD, st, [&] {
          return launch_gather_dfeats(net->bf16, L0.grad, L0.Cp, net->perm, net->n, net->d.c_in, d_dfeats, st);
        }) != hipSuccess)
      return SSCN_ERR_HIP;
  }
  // every weight gradient, the softmax layer's included, as one group
  WGradArgs w[MAX_WG_LAYERS];
  int nw = 0;
  for (int s = 1; s <= top; ++s)
    if (net->L[s].kind == 1) w[nw++] = conv_wgrad_args(net, s);
  {
    WGradArgs& f = w[nw++];
    f = WGradArgs{};
    const bool hd = head_drop(net).on;  // the softmax layer read its dropped input
    f.src = hd ? net->hdrop : Lt.X;
    f.src_stride = Lt.Cp;
    f.rmap = hd ? nullptr : net->head_rows;
    f.A = 1;
    f.cseg = Lt.Cp;
    f.m_ones = P.m_ones;
    f.Mpad = P.Mpad_w;
    f.dsrc = net->dlogits;
    f.dsrc_stride = net->dl_stride;
    f.dsrc_cols = net->dl_stride;
    f.Npad = P.Npad_w;
    f.rows_host = net->batch;
    f.nchunks = 1;
    f.slabs = 1;
    f.part = net->wpart;
    f.cfg = P.bn_w == 128 ? 0 : 1;
    f.dW = h_dW[fc];
    f.db = h_db[fc];
    f.c_in = P.c_in;
    f.c_out = P.c_out;
  }
  // (w[0] is the first convolution's, which the deferred final pass must precede)
  if (run_wgrads(net, w, nw, st, &deferred_fin, 0) != hipSuccess) return SSCN_ERR_HIP;
  net->backwarded = true;
  return SSCN_OK;
}

sscn_status sscn_set_dropout(sscn_net* net, const double* h_rates, int32_t n_rates, uint64_t seed) {
  if (!net) return SSCN_ERR_INVALID_ARGUMENT;
  if (n_rates == 0) {
    net->n_rates = 0;
    net->forwarded = false;
    return SSCN_OK;
  }
  if (!h_rates || n_rates != net->d.ell + 2) return SSCN_ERR_INVALID_ARGUMENT;
  bool any = false;
  for (int j = 0; j < n_rates; ++j) {
    if (!(h_rates[j] >= 0.0 && h_rates[j] < 1.0)) return SSCN_ERR_INVALID_ARGUMENT;
    any = any || h_rates[j] > 0.0;
  }
  if (any && !net->d.dropout) return SSCN_ERR_INVALID_ARGUMENT;
  for (int j = 0; j < n_rates; ++j) net->rates[j] = h_rates[j];
  net->n_rates = n_rates;
  net->seed = seed;
  net->forwarded = false;  // a backward pass must follow a forward pass with the same masks
  return SSCN_OK;
}

void sscn_philox4x32_10(const uint32_t counter[4], const uint32_t key[2], uint32_t out[4]) {
  if (!counter || !key || !out) return;
  const Philox4 r = philox4x32_10(counter[0], counter[1], counter[2], counter[3], key[0], key[1]);
  for (int e = 0; e < 4; ++e) out[e] = r.w[e];
}

sscn_status sscn_sgd_step(sscn_net* net, float* const* h_W32, void* const* h_W, float* const* h_b,
                          float* const* h_vW, float* const* h_vb, float lr, float momentum, float weight_decay,
                          void* stream) {
  if (!net || !h_W32 || !h_b || !h_vW || !h_vb) return SSCN_ERR_INVALID_ARGUMENT;
  if (!(lr >= 0.f) || !(momentum >= 0.f) || !(weight_decay >= 0.f) || !std::isfinite(lr) ||
      !std::isfinite(momentum) || !std::isfinite(weight_decay))
    return SSCN_ERR_INVALID_ARGUMENT;
  if (!net->backwarded) return SSCN_ERR_BAD_STATE;
  SgdArgs a;
  std::memset(&a, 0, sizeof(a));
  a.store_bf16 = net->bf16 ? 1 : 0;
  a.lr = lr;
  a.momentum = momentum;
  int blocks = 0;
  auto add = [&](float* w, void* ws, const float* g, float* v, int64_t n, float wd) {
    SgdJob& J = a.job[a.njobs];
    J.w = w;
    J.w_store = (ws == (void*)w) ? nullptr : ws;
    J.g = g;
    J.v = v;
    J.n = n;
    J.wd = wd;
    a.blk_beg[a.njobs] = blocks;
    blocks += (int)std::max<int64_t>(1, std::min<int64_t>(2048, (n + 255) / 256));
    ++a.njobs;
  };
  for (int p = 0; p < net->nparams; ++p) {
    const ParamPlan& P = net->P[p];
    if (!h_W32[p] || !h_b[p] || !h_vW[p] || !h_vb[p]) return SSCN_ERR_INVALID_ARGUMENT;
    void* store = h_W ? h_W[p] : nullptr;
    if (net->bf16 && !store) return SSCN_ERR_INVALID_ARGUMENT;  // the forward reads the bf16 copy
    add(h_W32[p], store, net->dW[p], h_vW[p], (int64_t)P.A * P.c_in * P.c_out, weight_decay);
    add(h_b[p], nullptr, net->db[p], h_vb[p], P.c_out, 0.f);
  }
  a.blk_beg[a.njobs] = blocks;
  return timed(net, SSCN_KC_SGD, (hipStream_t)stream, [&] { return launch_sgd(a, (hipStream_t)stream); }) ==
                 hipSuccess
             ? SSCN_OK
             : SSCN_ERR_HIP;
}

static size_t encode_bytes(int64_t N, int64_t batch, int64_t max_sites, size_t* offs) {
  const int64_t Wd = (N + 63) / 64;
  const int64_t words = batch * N * Wd;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = (off + 255) / 256 * 256;
    off = o + bytes;
    return o;
  };
  offs[0] = take(words * 8);            // bits
  offs[1] = take(words * 4);            // wpre
  offs[2] = take(batch * 4);            // scount
  offs[3] = take(batch * 4);            // soff
  offs[4] = take(4);                    // total
  offs[5] = take(4);                    // err
  offs[6] = take(max_sites * 8 * 4);    // counts
  return off + 256;
}

static bool encode_dims_ok(int32_t N, int32_t batch, int32_t max_sites) {
  return N >= 1 && N <= (3 << 8) && batch >= 0 && max_sites >= 0 && (int64_t)batch * N * N < (1ll << 31);
}

sscn_status sscn_encode_workspace_bytes(int32_t N, int32_t batch_max, int32_t max_sites, size_t* bytes) {
  if (!bytes || !encode_dims_ok(N, batch_max, max_sites)) return SSCN_ERR_INVALID_ARGUMENT;
  size_t offs[7];
  *bytes = encode_bytes(N, batch_max, max_sites, offs);
  return SSCN_OK;
}

}  // extern "C"

// The scratch of sscn_encode_strokes_static: one copy per GPU (a device
// variable of this code object), held until the process ends.  Host code never
// uses its name as an address: static_scratch() returns the device address
// taken with hipGetSymbolAddress on each device once.
static __device__ __align__(256) unsigned char scratch[SSCN_ENCODE_STATIC_SCRATCH_BYTES];

static void* static_scratch() {
  constexpr int MAX_DEVICES = 64;
  static std::mutex mu;
  static void* ptr[MAX_DEVICES] = {};
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  if (!ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    ptr[dev] = p;
  }
  return ptr[dev];
}

static sscn_status encode_strokes(int32_t N, int32_t dtype, const int32_t* d_points, int32_t n_points,
                                  const int32_t* d_stroke_begin, const int32_t* d_stroke_sample, int32_t n_strokes,
                                  int32_t batch, int32_t* d_coords, void* d_feats, int32_t max_sites,
                                  int32_t* h_count, void* d_ws, size_t ws_bytes, void* stream) {
  if (!h_count || !encode_dims_ok(N, batch, max_sites) || n_points < 0 || n_strokes < 0) return SSCN_ERR_INVALID_ARGUMENT;
  if (dtype != SSCN_F32 && dtype != SSCN_BF16) return SSCN_ERR_INVALID_ARGUMENT;
  if (!d_stroke_begin || (n_points > 0 && !d_points) || (n_strokes > 0 && !d_stroke_sample) ||
      (max_sites > 0 && (!d_coords || !d_feats)))
    return SSCN_ERR_INVALID_ARGUMENT;
  size_t offs[7];
  if (!d_ws || ((uintptr_t)d_ws & 255u) || ws_bytes < encode_bytes(N, batch, max_sites, offs))
    return SSCN_ERR_WORKSPACE;
  char* base = (char*)d_ws;
  EncodeArgs a;
  std::memset(&a, 0, sizeof(a));
  a.points = d_points;
  a.begin = d_stroke_begin;
  a.sample = d_stroke_sample;
  a.n_points = n_points;
  a.n_strokes = n_strokes;
  a.batch = batch;
  a.N = N;
  a.Wd = (N + 63) / 64;
  a.max_sites = max_sites;
  a.bits = (uint64_t*)(base + offs[0]);
  a.wpre = (int32_t*)(base + offs[1]);
  a.scount = (int32_t*)(base + offs[2]);
  a.soff = (int32_t*)(base + offs[3]);
  a.total = (int32_t*)(base + offs[4]);
  a.err = (int32_t*)(base + offs[5]);
  a.counts = (int32_t*)(base + offs[6]);
  a.coords = d_coords;
  hipStream_t st = (hipStream_t)stream;
  if (launch_encode(dtype == SSCN_BF16, a, d_feats, st) != hipSuccess) return SSCN_ERR_HIP;
  int32_t res[2] = {0, 0};
  if (hipMemcpyAsync(&res[0], a.total, 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipMemcpyAsync(&res[1], a.err, 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return SSCN_ERR_HIP;
  *h_count = res[0];
  if (res[1] & ERRBIT_ORDER) return SSCN_ERR_INVALID_ARGUMENT;
  if (res[1] & ERRBIT_RANGE) return SSCN_ERR_OUT_OF_RANGE;
  if (res[0] > max_sites) return SSCN_ERR_CAPACITY;
  return SSCN_OK;
}

extern "C" {

sscn_status sscn_encode_strokes(int32_t N, int32_t dtype, const int32_t* d_points, int32_t n_points,
                                const int32_t* d_stroke_begin, const int32_t* d_stroke_sample, int32_t n_strokes,
                                int32_t batch, int32_t* d_coords, void* d_feats, int32_t max_sites, int32_t* h_count,
                                void* d_ws, size_t ws_bytes, void* stream) {
  return encode_strokes(N, dtype, d_points, n_points, d_stroke_begin, d_stroke_sample, n_strokes, batch, d_coords,
                        d_feats, max_sites, h_count, d_ws, ws_bytes, stream);
}

sscn_status sscn_encode_strokes_static(int32_t N, int32_t dtype, const int32_t* d_points, int32_t n_points,
                                       const int32_t* d_stroke_begin, const int32_t* d_stroke_sample,
                                       int32_t n_strokes, int32_t batch, int32_t* d_coords, void* d_feats,
                                       int32_t max_sites, int32_t* h_count, void* stream) {
  if (!h_count || !encode_dims_ok(N, batch, max_sites)) return SSCN_ERR_INVALID_ARGUMENT;
  size_t offs[7];
  if (encode_bytes(N, batch, max_sites, offs) > SSCN_ENCODE_STATIC_SCRATCH_BYTES) return SSCN_ERR_WORKSPACE;
  void* ws = static_scratch();
  if (!ws) return SSCN_ERR_HIP;
  return encode_strokes(N, dtype, d_points, n_points, d_stroke_begin, d_stroke_sample, n_strokes, batch, d_coords,
                        d_feats, max_sites, h_count, ws, SSCN_ENCODE_STATIC_SCRATCH_BYTES, stream);
}

sscn_status sscn_forward_stage(sscn_net* net, int32_t stage, void* stream) {
  if (!net || stage < 1 || stage >= net->nlayers) return SSCN_ERR_INVALID_ARGUMENT;
  if (!net->forwarded) return SSCN_ERR_BAD_STATE;
  return forward_stage(net, stage, (hipStream_t)stream) == hipSuccess ? SSCN_OK : SSCN_ERR_HIP;
}

sscn_status sscn_backward_stage(sscn_net* net, int32_t stage, void* stream) {
  if (!net || stage < 1 || stage >= net->nlayers) return SSCN_ERR_INVALID_ARGUMENT;
  if (!net->forwarded || !net->dW[0]) return SSCN_ERR_BAD_STATE;
  hipStream_t st = (hipStream_t)stream;
  hipError_t e;
  if (net->L[stage].kind == 1) {
    // delta of this layer as it stands: its own sums, weight gradient, gradient below
    const WGradArgs w = conv_wgrad_args(net, stage);
    if ((e = ground_level(net, stage, false, st)) == hipSuccess && (e = run_wgrads(net, &w, 1, st)) == hipSuccess)
      e = rows_below(net, stage, st);
  } else {
    // rows >= 1 below, then row 0 below with the sums of the convolution below
    if ((e = rows_below(net, stage, st)) == hipSuccess) e = ground_level(net, stage - 1, true, st);
  }
  return e == hipSuccess ? SSCN_OK : SSCN_ERR_HIP;
}

sscn_status sscn_timing_enable(sscn_net* net, uint32_t class_mask) {
  if (!net) return SSCN_ERR_INVALID_ARGUMENT;
  net->tmask = class_mask & ((1u << SSCN_KC_COUNT) - 1u);
  return SSCN_OK;
}

sscn_status sscn_timing_collect(sscn_net* net, int32_t kernel_class, int32_t* launches, float* total_ms,
                                void* stream) {
  if (!net || !launches || !total_ms || kernel_class < 0 || kernel_class >= SSCN_KC_COUNT)
    return SSCN_ERR_INVALID_ARGUMENT;
  if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return SSCN_ERR_HIP;
  int32_t n = 0;
  float tot = 0.f;
  std::vector<sscn_net::Rec> keep;
  for (const auto& r : net->recs) {
    if (r.cls != kernel_class) {
      keep.push_back(r);
      continue;
    }
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return SSCN_ERR_HIP;
    tot += ms;
    ++n;
  }
  net->recs.swap(keep);
  if (net->recs.empty()) net->ev_next = 0;
  *launches = n;
  *total_ms = tot;
  return SSCN_OK;
}

sscn_status sscn_timing_launches(sscn_net* net, int32_t kernel_class, int32_t* h_tags, float* h_ms,
                                 int32_t capacity, int32_t* count, void* stream) {
  if (!net || !count || kernel_class < 0 || kernel_class >= SSCN_KC_COUNT || capacity < 0 ||
      (capacity > 0 && (!h_tags || !h_ms)))
    return SSCN_ERR_INVALID_ARGUMENT;
  if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return SSCN_ERR_HIP;
  int32_t n = 0;
  std::vector<sscn_net::Rec> keep;
  for (const auto& r : net->recs) {
    if (r.cls != kernel_class) {
      keep.push_back(r);
      continue;
    }
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return SSCN_ERR_HIP;
    if (n < capacity) {
      h_tags[n] = r.tag;
      h_ms[n] = ms;
    }
    ++n;
  }
  net->recs.swap(keep);
  if (net->recs.empty()) net->ev_next = 0;
  *count = n;
  return SSCN_OK;
}

sscn_status sscn_layer_view_get(const sscn_net* net, int32_t layer, sscn_layer_view* out) {
  if (!net || !out || layer < 0 || layer >= net->nlayers) return SSCN_ERR_INVALID_ARGUMENT;
  if (!net->ws) return SSCN_ERR_BAD_STATE;
  const LayerPlan& L = net->L[layer];
  out->kind = L.kind;
  out->side = L.S;
  out->channels = L.C;
  out->row_stride = L.Cp;
  out->window = layer ? L.A : 0;
  out->capacity = (int32_t)L.cap;
  out->count = net->counts + layer;
  out->sites = L.sites;
  out->rules = L.rules;
  out->rules_t = L.rules_t;
  out->features = L.X;
  out->grad = L.grad;
  out->argmax = L.argmax;
  out->gmask = L.gmask;
  return SSCN_OK;
}

}  // extern "C"
