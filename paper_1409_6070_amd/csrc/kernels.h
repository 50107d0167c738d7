// Host-side launchers of the HIP kernels (internal to libsscn).
#pragma once

#include <algorithm>

#include "common.h"

namespace sscn {

struct SitesWork {
  int64_t total;
  int64_t base[MAX_LAYERS + 1];
};

hipError_t launch_rulebook(const RulebookArgs& a, const SitesWork& wk, int32_t max_words, hipStream_t st);

// ---------------------------------------------------------------------------
// gather GEMM: out[m][n] = epi( sum_k A(m,k) * Bt[n][k] ),
//   A(m, k) = src[rmap[m*A + f]][c] with k = f*cseg + c   (rmap entry -1: zero;
//   rmap null: source row m, A must be 1)

enum Epilogue : int32_t {
  EPI_BIAS_RELU = 0,  // + bias, ReLU, store in storage dtype
  EPI_BIAS_F32 = 1,   // + bias, store float32
  EPI_F32 = 2,        // store float32
  EPI_STORE = 3,      // store in storage dtype
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
};

// weight-gradient GEMM, split over sites:
//   part[chunk][m][n] = sum_{o in chunk} A(o, m) * dsrc[o][n]
//   A(o, m) = src[rmap[o*A + f]][c] for m = f*cseg + c < A*cseg;
//   A(o, m_ones) = 1;  A(o, m_ind + f) = [rmap[o*A + f] == 0]
struct WGradArgs {
  const void* src;
  int32_t src_stride;
  const int32_t* rmap;
  int32_t A;
  int32_t cseg;
  int32_t m_ones;
  int32_t m_ind;
  int32_t Mpad;
  const void* dsrc;
  int32_t dsrc_stride;
  int32_t dsrc_cols;
  int32_t Npad;
  const int32_t* rows_dev;
  int32_t rows_add;
  int32_t rows_host;
  int32_t nchunks;
  float* part;
};

struct GemmTile {
  int BM, BN, BK;
};
GemmTile gemm_tile(bool bf16);

hipError_t launch_gemm(bool bf16, const GemmArgs& a, int64_t max_rows, hipStream_t st);
hipError_t launch_wgrad(bool bf16, const WGradArgs& a, hipStream_t st);

// part -> dW [A*c_in x c_out], db [c_out], D0 [A x c_out] (ground-row sums)
hipError_t launch_wgrad_reduce(const float* part, int32_t nchunks, int32_t Mpad, int32_t Npad, int32_t A, int32_t cseg,
                               int32_t c_in, int32_t c_out, int32_t m_ones, int32_t m_ind, float* dW, float* db,
                               float* D0, hipStream_t st);
// grad_in[0][c] = sum_f sum_n W[(f*c_in + c)*c_out + n] * D0[f][n]
hipError_t launch_row0_dx(bool bf16, const void* W, const float* D0, int32_t A, int32_t c_in, int32_t c_out,
                          int32_t cp_in, void* grad_in, hipStream_t st);

// ---------------------------------------------------------------------------
// max-pooling

hipError_t launch_pool_fwd(bool bf16, const void* X_in, int32_t stride_in, const int32_t* R, void* X_out,
                           int32_t stride_out, uint8_t* argmax, int32_t cp, const int32_t* n_out, int64_t cap_out,
                           hipStream_t st);
// routes dY back to the rows below and applies the ReLU mask of the convolution below
hipError_t launch_pool_bwd(bool bf16, const void* dY, int32_t stride, const uint8_t* argmax, const int32_t* Pt,
                           const int32_t* R, const void* Y_below, void* grad_below, int32_t cp, const int32_t* n_out,
                           const int32_t* n_in, int64_t cap_in, int64_t cap_out, float* part, int32_t nparts,
                           hipStream_t st);

// ---------------------------------------------------------------------------
// input, parameters, head

hipError_t launch_scatter_input(bool bf16, const void* feats, int32_t n, int32_t c_in, const int32_t* perm, void* X0,
                                int32_t cp0, hipStream_t st);
hipError_t launch_gather_dfeats(bool bf16, const void* grad0, int32_t cp0, const int32_t* perm, int32_t n,
                                int32_t c_in, void* dfeats, hipStream_t st);
// Bt[n][k] = (n < rows_n && k-map valid) ? W[...] : 0, for the two packings
//   mode 0 (forward):   Bt[n][f*cp_in + c]  = W[(f*c_in + c)*c_out + n]
//   mode 1 (backward):  Bt[c][f*cp_out + n] = W[(f*c_in + c)*c_out + n]
hipError_t launch_pack(bool bf16, int mode, const void* W, int32_t A, int32_t c_in, int32_t c_out, int32_t cp_in,
                       int32_t cp_out, void* Bt, int32_t Npad, int32_t Kpad, hipStream_t st);
hipError_t launch_softmax_xent(bool bf16, const float* logits, const int32_t* labels, int32_t batch, int32_t classes,
                               void* dlogits, int32_t dl_stride, float* loss_part, float* loss, hipStream_t st);
hipError_t launch_head_scatter(bool bf16, const float* dh, int32_t dh_stride, const int32_t* head_rows,
                               int32_t batch, const void* Y_top, void* grad_top, int32_t cp, hipStream_t st);
hipError_t launch_fill_zero(void* p, int64_t bytes, hipStream_t st);

}  // namespace sscn
