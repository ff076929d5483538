/*
 * surge_ops.h - stage-level entry points of the SuperBatch encoder.
 *
 * Each call runs one stage of the encode path on caller-provided device
 * buffers, with the same kernels surge_encode_superbatch launches, so every
 * stage can be checked on its own.  The call is synchronous: it enqueues on
 * `hip_stream` (NULL = null stream) and waits for it before returning.
 * bf16 tensors are passed as uint16_t bit patterns.  Text boundaries are
 * given as host int64 cu_seqlens [n_texts+1] (cu[0] = 0, increasing), checked
 * on the host and copied to the device by the call.  Returns the status
 * codes of surge.h.
 */
#ifndef SURGE_OPS_H_
#define SURGE_OPS_H_

#include <stdint.h>

#include "surge.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Embedding gather + LayerNorm (encoder input; positions restart at 0 for
 * every text): out[t] = LN(word[id_t] + pos[t - cu_i]).
 * d_tokens int32 [cu[n]]; d_word bf16 [vocab, d]; d_pos bf16 [max_pos, d];
 * gamma/beta fp32 [d]; d_out bf16 [cu[n], d].  d % 128 == 0, d <= 1024,
 * every text length <= min(max_pos, 4096).  Out-of-vocabulary IDs are read
 * as ID 0 and reported with SURGE_ERR_INVALID_ARGUMENT after the stage ran.
 */
surge_status surge_op_embed_ln(int64_t n_texts, const int64_t* h_cu_seqlens, const int32_t* d_tokens,
                               const uint16_t* d_word, int32_t vocab, const uint16_t* d_pos,
                               int32_t max_pos, const float* d_gamma, const float* d_beta,
                               float eps, int32_t d, uint16_t* d_out, void* hip_stream);

/*
 * Linear layer over packed tokens: Y = epi(X W^T + b).
 * d_x bf16 [M, K]; d_w bf16 [N, K] (out, in); d_bias fp32 [N];
 * epilogue 0 = bias, 1 = bias then exact GELU, 2 = bias then + d_res
 * (bf16 [M, N]); d_y bf16 [M, N].  M >= 1, N % 128 == 0, K % 64 == 0.
 */
surge_status surge_op_linear(int64_t M, int32_t N, int32_t K, const uint16_t* d_x,
                             const uint16_t* d_w, const float* d_bias, const uint16_t* d_res,
                             int32_t epilogue, uint16_t* d_y, void* hip_stream);

/*
 * The linear layer's LayerNorm-fused forms (post-LN encoder with every
 * LayerNorm except the last folded into its neighbours; LN(v) = gamma (v -
 * mu) / sqrt(var + eps) + beta over a row, biased variance):
 *   epilogue 3: y = LN(x) W^T + b for raw rows x of d_x, computed as
 *               rstd (x W'^T - mu s) + b' with d_w = W' = bf16(W diag(gamma)),
 *               d_col_s = s = row sums of W' [N] and d_bias = b' = b + W beta;
 *               the row statistics of x come from d_stats_in;
 *   epilogue 4: epilogue 3, then exact GELU;
 *   epilogue 5: y = x W^T + b + res, and the statistics of y's rows are
 *               written to d_stats_out;
 *   epilogue 6: y = x W^T + b + LN(res) with res's statistics in d_stats_in
 *               and LN's gamma, beta in d_gamma, d_beta [N]; statistics of y
 *               to d_stats_out.
 *   epilogues 0-2 as surge_op_linear.
 * Statistics are partials of W = surge_op_linear_stats_width(M, N) (64)
 * consecutive features of a row: fp32 pairs (mean, variance) at
 * [(p * M + row) * 2], p < N / W.  d_stats_in holds parts_in partials of
 * equal width per row (the producer's N / W).  Shapes as surge_op_linear;
 * float vectors 16-byte aligned.
 */
surge_status surge_op_linear_ln(int64_t M, int32_t N, int32_t K, const uint16_t* d_x,
                                const uint16_t* d_w, const float* d_bias, const uint16_t* d_res,
                                int32_t epilogue, const float* d_stats_in, int32_t parts_in,
                                const float* d_col_s, const float* d_gamma, const float* d_beta,
                                float eps, float* d_stats_out, uint16_t* d_y, void* hip_stream);

/*
 * surge_op_linear_ln without any allocation, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the per-row LayerNorm factors that the
 * folded and residual-LayerNorm epilogues (3, 4, 6) read live in a static
 * device array of the library (4 MiB: at most 524,288 rows), not in a buffer
 * allocated per call.  Same arguments, checks, kernels and results as
 * surge_op_linear_ln, but asynchronous: the call only enqueues on
 * `hip_stream` (no synchronisation).  M above 524,288 with epilogue 3, 4 or
 * 6 returns SURGE_ERR_CAPACITY before anything is enqueued.  Every call on
 * one GPU shares that GPU's array (each call overwrites the rows it uses
 * before reading them): calls on one stream are ordered, calls that overlap
 * on different streams of one GPU race.  Calls no hipMalloc/hipFree.
 */
surge_status surge_op_linear_ln_noalloc(int64_t M, int32_t N, int32_t K, const uint16_t* d_x,
                                        const uint16_t* d_w, const float* d_bias,
                                        const uint16_t* d_res, int32_t epilogue,
                                        const float* d_stats_in, int32_t parts_in,
                                        const float* d_col_s, const float* d_gamma,
                                        const float* d_beta, float eps, float* d_stats_out,
                                        uint16_t* d_y, void* hip_stream);

/* Features per statistics partial of an [M, N] linear output (host-only). */
int32_t surge_op_linear_stats_width(int64_t M, int32_t N);

/*
 * Packed varlen multi-head self-attention within each text:
 * out[rows of text i, head h] = softmax(Q_h K_h^T / sqrt(d_head)) V_h.
 * d_qkv bf16 [T, 3 n_heads d_head] (Q | K | V blocks, head h at columns
 * h d_head of each); d_out bf16 [T, n_heads d_head]; T = cu[n_texts].
 * d_head is 32 or 64; n_heads * d_head % 128 == 0; every text length in
 * [1, 4096].
 */
surge_status surge_op_attention(int64_t n_texts, const int64_t* h_cu_seqlens, int32_t n_heads,
                                int32_t d_head, const uint16_t* d_qkv, uint16_t* d_out,
                                void* hip_stream);

/* Row LayerNorm: y = gamma (x - mean) / sqrt(var + eps) + beta, biased
 * variance.  d_x, d_y bf16 [M, d]; d % 8 == 0, d <= 1024. */
surge_status surge_op_layernorm(int64_t M, int32_t d, const uint16_t* d_x, const float* d_gamma,
                                const float* d_beta, float eps, uint16_t* d_y, void* hip_stream);

/* Masked mean pooling + L2 normalisation: out[i] = e_i / max(||e_i||, 1e-12)
 * with e_i the mean of text i's rows of d_x (bf16 [T, d]); d_out fp32
 * [n_texts, d], 16-byte aligned.  d % 128 == 0, d <= 1024. */
surge_status surge_op_pool_l2(int64_t n_texts, const int64_t* h_cu_seqlens, int32_t d,
                              const uint16_t* d_x, float* d_out, void* hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* SURGE_OPS_H_ */
