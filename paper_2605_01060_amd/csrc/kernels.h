// Host-side launchers of the gfx950 kernels.  Every launcher assumes its
// arguments were checked by the caller (shapes, alignment, index ranges) and
// returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace surge {

// x_t = LN(word[id_t] + pos[t - cu_i]) for every token.  tokens [T],
// cu int32 [n_texts+1] and the row_block_items work items (device), one
// workgroup per item; out bf16 [T, d].  Out-of-vocabulary IDs are gathered
// as ID 0 and set *err = 1.
hipError_t launch_embed_ln(const int32_t* tokens, const int32_t* cu, const uint32_t* items,
                           int n_items, const uint16_t* word, const uint16_t* pos,
                           const float* gamma, const float* beta, float eps, int vocab, int d,
                           uint16_t* out, int* err, hipStream_t stream);

// Y[M, N] = epi(X[M, K] W^T + b), W stored [N, K] (out, in), bf16 in/out.
// Requires N % 128 == 0, K % 64 == 0, M >= 1.
//   EPI_BIAS          y = acc + b
//   EPI_BIAS_GELU     y = GELU(acc + b)
//   EPI_BIAS_RESIDUAL y = acc + b + R
// LayerNorm folded into its neighbours (post-LN encoder, LN(x) = g (x - mu)
// rstd + beta per row of x):
//   EPI_FOLD          X holds raw rows x (K features) whose per-row
//                     LayerNorm factors are in ex.rows_in; W was built as W diag(g)
//                     and b as b + W beta, and ex.col_s[n] = sum_k W'[n][k],
//                     so y = rstd (acc - mu col_s) + b = LN(x) W^T + b;
//   EPI_FOLD_GELU     the same, then GELU;
//   EPI_RES_STATS     y = acc + b + R, and the per-row statistics of y go
//                     to ex.stats_out;
//   EPI_LNRES_STATS   y = acc + b + LN(R) with R's LayerNorm factors in
//                     ex.rows_in and LN's g, beta in ex.gamma, ex.beta; the
//                     statistics of y go to ex.stats_out.
// Row statistics are partials over linear_stats_width(M, N) = 64
// consecutive features in every tile configuration: float2 (mean, variance)
// at [p * M + row], p < N / 64;
// launch_ln_rows turns them into the per-row LayerNorm factors
// float2 (rstd, -mean * rstd) at [row].
enum LinearEpilogue {
  EPI_BIAS = 0,
  EPI_BIAS_GELU = 1,
  EPI_BIAS_RESIDUAL = 2,
  EPI_FOLD = 3,
  EPI_FOLD_GELU = 4,
  EPI_RES_STATS = 5,
  EPI_LNRES_STATS = 6,
};
struct LinearExtra {
  const float2* rows_in = nullptr;   // LayerNorm factors of X's rows (FOLD) or R's rows (LNRES)
  float2* stats_out = nullptr;       // partials of Y's rows (RES_STATS, LNRES_STATS)
  const float* col_s = nullptr;      // [N] (FOLD)
  const float* gamma = nullptr;      // [N] (LNRES)
  const float* beta = nullptr;       // [N] (LNRES)
  int n_cus = 0;                     // compute units of the device (0: query it)
};
hipError_t launch_linear(const uint16_t* X, const uint16_t* W, const float* bias, const uint16_t* R,
                         uint16_t* Y, int64_t M, int N, int K, int epi, const LinearExtra& ex,
                         hipStream_t stream);
// Features per statistics partial written by launch_linear for an [M, N]
// output (the width of one wave's slice of a tile).
int linear_stats_width(int64_t M, int N);

// Packed varlen multi-head self-attention.  qkv bf16 [T, 3 H dh] (Q | K | V
// column blocks, head h at columns h*dh of each), out bf16 [T, H dh].
// Attention runs within each text only.  dh is 32 or 64.  items lists the
// (text << 7 | 32-row block) work items built by row_block_items.
hipError_t launch_attention(const uint16_t* qkv, uint16_t* out, const int32_t* cu,
                            const uint32_t* items, int n_items, int n_heads, int d_head,
                            hipStream_t stream);

// Work items of a chunk: (text << 7 | block) for every block of 32
// consecutive rows of a text (the attention's query blocks, the
// embedding's row blocks); at most cu[n_texts] of them, every text length
// in [1, 4096]; longest text first.  Returns the item count.
int row_block_items(const int64_t* cu, int64_t n_texts, uint32_t* items);

// Per-row LayerNorm factors rows[m] = (rstd, -mean * rstd) from `parts`
// equal-width statistics partials stats[p * M + m] = (mean, variance).
hipError_t launch_ln_rows(const float2* stats, int parts, int64_t M, float eps, float2* rows,
                          hipStream_t stream);

// y = LN(x) per row of d (d % 8 == 0, d <= 1024), bf16 in/out.
hipError_t launch_layernorm(const uint16_t* x, const float* gamma, const float* beta, float eps,
                            uint16_t* y, int64_t M, int d, hipStream_t stream);

// e_i = mean of text i's rows of x; row i of the output (dst[i], a device
// pointer to d floats) = e_i / max(||e_i||, 1e-12).  With rows != NULL the
// rows of x are raw and LayerNorm(gamma, beta) is applied to each first,
// from its factors rows[t] = (rstd, -mean * rstd).
hipError_t launch_pool_l2_scatter(const uint16_t* x, const int32_t* cu, int n_texts,
                                  const uint64_t* dst, int d, const float2* rows,
                                  const float* gamma, const float* beta, hipStream_t stream);

}  // namespace surge
