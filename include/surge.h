/*
 * surge.h - C-ABI of the SuperBatch encoder for MI355X (gfx950).
 *
 * SURGE (arXiv 2605.01060) groups many small logical partitions of texts into
 * SuperBatches and encodes each SuperBatch with a single call (Alg. 1,
 * Flush), slicing the embedding matrix back per partition.  This library is
 * that encode call on one GPU: many short, variable-length texts packed back
 * to back without padding, a post-LN BERT-style encoder, masked mean pooling,
 * L2 normalisation and a scatter of every text's row into its partition's
 * output segment.
 *
 * Problem statement (Sec. 2.2): partitions (k_i, T_i), n_i texts each,
 * sum n_i = N; the output gives every partition an fp32 matrix E_i of shape
 * [n_i, d], row r being the embedding of the partition's r-th text.
 *
 * Conventions shared by every entry point:
 *   - Partition p's texts are the global texts part_offsets[p] ..
 *     part_offsets[p+1]-1 (CSR, partitions in arrival order, Alg. 1's
 *     "ordered by key" precondition).
 *   - Tokens are int32 IDs packed back to back; text i owns tokens
 *     cu_seqlens[i] .. cu_seqlens[i+1]-1.  There is no padding and no mask.
 *   - "host" pointers are CPU memory read before the call returns (the
 *     library copies what it needs); "device" pointers are GPU memory that
 *     must stay valid and unmodified until the stream has passed the work
 *     the call enqueued.  The caller owns every buffer and the stream.
 *   - Every argument check is done on the host before anything is enqueued:
 *     a call that returns an error has written no output byte.
 *   - Calls return SURGE_OK or an error code; surge_last_error() gives a
 *     message (thread-local, valid until the next call on that thread).
 *   - An encoder is not thread-safe: use one encoder per host thread.  Its
 *     device workspace is shared by every call, so each encode call first
 *     makes its stream(s) wait for the previous call's work (on whatever
 *     stream that ran): calls on different streams are ordered, never
 *     overlapped, without any host synchronisation.
 */
#ifndef SURGE_H_
#define SURGE_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t surge_status;
#define SURGE_OK 0
#define SURGE_ERR_INVALID_ARGUMENT 1 /* a malformed argument; nothing enqueued */
#define SURGE_ERR_CAPACITY 2         /* an output array is too small */
#define SURGE_ERR_OUT_OF_MEMORY 3    /* device or pinned allocation failed */
#define SURGE_ERR_DEVICE 4           /* a HIP runtime call failed */
#define SURGE_ERR_INTERNAL 5

/* SuperBatch formation policies (Alg. 1 and its two readings). */
#define SURGE_POLICY_SPLIT 0   /* pre-append cap flush + split of oversized
                                  partitions (Sec. 3.2 prose, Sec. 6) */
#define SURGE_POLICY_LITERAL 1 /* Alg. 1 as printed: append, then flush on
                                  total >= cap or total >= b_min */

/* Element type of the host weight arrays given to surge_encoder_create. */
#define SURGE_WEIGHTS_F32 0  /* IEEE float32 */
#define SURGE_WEIGHTS_BF16 1 /* bfloat16 bit patterns (uint16_t), e.g. a bf16 checkpoint */

/* Shape of a post-LN BERT-style encoder.  d_model % n_heads == 0 and
 * d_model / n_heads is 32 or 64; d_model and d_ff are multiples of 128. */
typedef struct surge_encoder_desc {
  int32_t n_layers;
  int32_t d_model;
  int32_t n_heads;
  int32_t d_ff;
  int32_t vocab_size;
  int32_t max_positions; /* longest text, in tokens */
  float ln_eps;          /* LayerNorm epsilon (1e-12 for BERT) */
  int32_t weight_dtype;  /* SURGE_WEIGHTS_F32 or SURGE_WEIGHTS_BF16 */
} surge_encoder_desc;

/* One bound of a SuperBatch (Alg. 1, Flush: (start, end, key)): texts
 * first_text .. first_text+count-1 are rows row_offset .. row_offset+count-1
 * of partition `partition`.  row_offset is non-zero only for the later
 * pieces of a partition split across SuperBatches (Sec. 6). */
typedef struct surge_segment {
  int64_t first_text;
  int64_t count;
  int64_t row_offset;
  int32_t partition;
  int32_t reserved;
} surge_segment;

/* One SuperBatch: global texts text_begin .. text_end-1, described by
 * segments seg_begin .. seg_end-1 of the segment array. */
typedef struct surge_superbatch {
  int64_t text_begin;
  int64_t text_end;
  int64_t seg_begin;
  int64_t seg_end;
} surge_superbatch;

typedef struct surge_encoder surge_encoder; /* opaque */

/* Library version, "major.minor.patch". */
const char* surge_version(void);

/* Message of the last failed call on this thread ("" if none). */
const char* surge_last_error(void);

/*
 * SuperBatch formation (Alg. 1, AddPartition / Flush; Sec. 3.2 two-threshold
 * scheme; Sec. 6 oversized partitions).  Pure host code, no GPU needed.
 *
 * part_offsets: host int64 [n_parts+1], part_offsets[0] = 0, non-decreasing.
 *   Empty partitions are allowed; they never reach AddPartition and produce
 *   no segment.
 * b_min: efficiency trigger, >= 1.  n_max: upper threshold in texts (B_max,
 *   the per-SuperBatch cap); <= 0 disables it.
 * policy: SURGE_POLICY_SPLIT or SURGE_POLICY_LITERAL.
 * sbs/segs: host output arrays of sb_cap / seg_cap entries.  With sbs and
 *   segs both NULL the call only counts (n_sbs, n_segs).  If a capacity is
 *   too small the call writes the counts, nothing else, and returns
 *   SURGE_ERR_CAPACITY.
 */
surge_status surge_plan(const int64_t* part_offsets, int32_t n_parts, int64_t b_min, int64_t n_max,
                        int32_t policy, surge_superbatch* sbs, int64_t sb_cap, int64_t* n_sbs,
                        surge_segment* segs, int64_t seg_cap, int64_t* n_segs);

/*
 * The host-side argument check of surge_encode_superbatch, exposed on its own
 * (pure host code, no GPU needed).  Checks: 0 <= n_texts; cu_seqlens[0] = 0,
 * every text length in [1, desc->max_positions], cu_seqlens[n_texts] =
 * n_tokens; the segments tile texts 0 .. n_texts-1 in order with count >= 1;
 * every partition index in [0, n_parts); every segment fits its partition
 * (row_offset >= 0, row_offset + count <= part_sizes[p]); part_out[p] is
 * non-NULL for every partition a segment writes.  Returns
 * SURGE_ERR_INVALID_ARGUMENT naming the first violation.
 */
surge_status surge_validate_superbatch(const surge_encoder_desc* desc, int64_t n_texts, int64_t n_tokens,
                                       const int64_t* h_cu_seqlens, const surge_segment* h_segs,
                                       int64_t n_segs, const int64_t* h_part_sizes,
                                       float* const* h_part_out, int32_t n_parts);

/*
 * The host-side argument check of the whole-input entry points
 * (surge_encode_all, surge_encode_all_streamed), exposed on its own (pure
 * host code, no GPU needed).  Plans the input with surge_plan(part_offsets,
 * n_parts, b_min, n_max, policy) and checks: part_offsets[n_parts] =
 * n_texts; cu_seqlens[0] = 0 and every text length in [1,
 * desc->max_positions]; every SuperBatch of the plan holds fewer than 2^31
 * tokens; part_out[p] is non-NULL for every non-empty partition.  The total
 * token count is not capped (offsets are int64 throughout).  Optionally
 * returns the plan's SuperBatch count and its largest SuperBatch in texts
 * and in tokens (any pointer may be NULL).
 */
surge_status surge_validate_input(const surge_encoder_desc* desc, int64_t n_texts,
                                  const int64_t* h_cu_seqlens, const int64_t* h_part_offsets,
                                  int32_t n_parts, int64_t b_min, int64_t n_max, int32_t policy,
                                  float* const* h_part_out, int64_t* n_superbatches,
                                  int64_t* max_sb_texts, int64_t* max_sb_tokens);

/*
 * Create an encoder on the current HIP device.
 *
 * host_weights: n_weights = 4 + 12 * n_layers host arrays of
 *   desc->weight_dtype elements (float32, or bf16 bit patterns), row-major, in
 *   this order: word_emb [vocab, d], pos_emb [max_positions, d], ln_e gamma
 *   [d], ln_e beta [d]; then per layer: W_qkv [d, 3d], b_qkv [3d], W_o [d, d],
 *   b_o [d], ln1 gamma [d], ln1 beta [d], W_1 [d, d_ff], b_1 [d_ff],
 *   W_2 [d_ff, d], b_2 [d], ln2 gamma [d], ln2 beta [d].  Matrices are
 *   [in, out] (y = x W + b); W_qkv holds Q | K | V as column blocks, head h
 *   owning columns [h*dh, (h+1)*dh) of each block.  Matrices and embedding
 *   tables are rounded to bf16 (nearest, ties to even; bf16 input is used
 *   as is); biases and LayerNorm parameters are kept in fp32 (bf16 input is
 *   widened exactly).  float32 arrays holding bf16-representable values and
 *   the bf16 arrays of the same values give bit-identical encoders.  The
 *   caller may free the host arrays when the call returns.
 * max_tokens_per_chunk: size of the activation workspace in tokens (>=
 *   max_positions).  A SuperBatch with more tokens is encoded in several
 *   chunks cut at text boundaries; results do not depend on the cut.
 */
surge_status surge_encoder_create(const surge_encoder_desc* desc, const void* const* host_weights,
                                  int32_t n_weights, int64_t max_tokens_per_chunk,
                                  surge_encoder** out);

/* Free the encoder's device memory.  Waits for its outstanding work. */
void surge_encoder_destroy(surge_encoder* enc);

/* The encoder's description and workspace size. */
surge_status surge_encoder_info(const surge_encoder* enc, surge_encoder_desc* desc,
                                int64_t* max_tokens_per_chunk, int64_t* workspace_bytes);

/*
 * Encode one SuperBatch (Alg. 1, Flush): embed, run the encoder over the
 * packed tokens, mean-pool and L2-normalise each text, and write each text's
 * row into its partition's segment.  Asynchronous on `hip_stream` (NULL =
 * the null stream).
 *
 * d_token_ids: device int32 [n_tokens], the SuperBatch's texts back to back.
 *   IDs outside [0, vocab) are replaced by 0 and reported by surge_check.
 * h_cu_seqlens: host int64 [n_texts+1], SuperBatch-local, cu[0] = 0.
 * h_segs/n_segs: the SuperBatch's bounds, first_text SuperBatch-local.
 * h_part_out: host array [n_parts] of device pointers; partition p's output
 *   is fp32 row-major [h_part_sizes[p], d_model].  Only the rows named by
 *   the segments are written, each exactly once.
 * n_texts = 0 is valid and enqueues nothing.
 */
surge_status surge_encode_superbatch(surge_encoder* enc, int64_t n_texts, int64_t n_tokens,
                                     const int32_t* d_token_ids, const int64_t* h_cu_seqlens,
                                     const surge_segment* h_segs, int64_t n_segs,
                                     float* const* h_part_out, const int64_t* h_part_sizes,
                                     int32_t n_parts, void* hip_stream);

/*
 * Encode a whole partition-grouped input: form the SuperBatches with
 * surge_plan(part_offsets, n_parts, b_min, n_max, policy) and encode
 * SuperBatches first_sb .. end in order (first_sb > 0 resumes a run at a
 * SuperBatch boundary; the plan is a deterministic function of its inputs).
 *
 * d_token_ids: device int32, all tokens, texts back to back (global).
 * h_cu_seqlens: host int64 [n_texts+1], global.
 * h_part_offsets: host int64 [n_parts+1]; part_offsets[n_parts] = n_texts.
 * h_part_out: host array [n_parts] of device pointers to fp32 [n_p, d].
 * n_superbatches: optional (may be NULL), receives the plan's SuperBatch count.
 */
surge_status surge_encode_all(surge_encoder* enc, int64_t n_texts, const int32_t* d_token_ids,
                              const int64_t* h_cu_seqlens, const int64_t* h_part_offsets,
                              int32_t n_parts, int64_t b_min, int64_t n_max, int32_t policy,
                              float* const* h_part_out, int64_t first_sb, int64_t* n_superbatches,
                              void* hip_stream);

/*
 * Timing of one streamed encode (surge_encode_all_streamed), from HIP events
 * on the two streams; milliseconds.  I/O here is the PCIe traffic either
 * side of the path: the upload of a SuperBatch's tokens and the download of
 * its embeddings (the GPU analogue of the paper's serialise + upload stage,
 * Sec. 3.3).
 */
typedef struct surge_stream_stats {
  int64_t n_superbatches;
  double total_ms;  /* start of the first upload -> end of the last download */
  double ttfo_ms;   /* start of the first upload -> end of SuperBatch 0's download */
  double enc_ms;    /* sum over SuperBatches of the encode span */
  double h2d_ms;    /* sum of the token uploads */
  double d2h_ms;    /* sum of the embedding downloads */
  /* I/O overlap ratio of eq. (overlap): 1 - max(0, t_io - t_enc) / t_io with
   * t_enc and t_io = t_h2d + t_d2h the per-SuperBatch means. */
  double rho;
  /* Measured counterpart: 1 - (total_ms - enc_ms) / (h2d_ms + d2h_ms), the
   * share of the I/O time that did not extend the wall time (clamped to
   * [0, 1]). */
  double rho_measured;
  /* Device staging memory the call allocated: two token buffers for the
   * plan's largest SuperBatch in tokens and (overlap 0 and 1) two embedding
   * buffers for its largest SuperBatch in texts, i.e. twice Lemma 1's
   * M(S) = S L + 4 S d with the text part as int32 token IDs (Sec. 4.3),
   * bounded through S <= B_min - 1 + n_max and, with the cap, S <= n_max. */
  int64_t staging_bytes;
  int64_t max_sb_texts;
  int64_t max_sb_tokens;
} surge_stream_stats;

/*
 * Encode a whole partition-grouped input that lives in host memory, as a
 * stream of SuperBatches (the plan of surge_plan with the same arguments):
 * SuperBatch j's tokens are uploaded, encoded and its embeddings downloaded
 * into h_out.  With overlap = 1 the uploads and downloads run on
 * `copy_stream`, double-buffered, so the download of SuperBatch j and the
 * upload of j+1 overlap the encode of j+1 on `compute_stream` (Sec. 3.3,
 * Alg. 2 on the PCIe side of the GPU).  With overlap = 0 everything runs on
 * `compute_stream` in order (the synchronous baseline).  With overlap = 2
 * (zero copy) the tokens are uploaded in order on `compute_stream` and the
 * pooling kernel writes every embedding straight into h_out through its
 * device mapping, so no download runs at all; h_out must then be pinned
 * host memory mapped for the device (hipHostMalloc) over all n_texts rows,
 * else SURGE_ERR_INVALID_ARGUMENT before anything runs, and the download
 * times read 0.  Returns after both streams have finished.  Zero copy is
 * the fastest of the three on MI355X: the runtime moves pinned-memory
 * copies with copy kernels that take compute units from the encode, so the
 * double-buffered overlap gains nothing over the in-order mode.
 *
 * h_token_ids: host int32 [h_cu_seqlens[n_texts]], texts back to back.
 * h_cu_seqlens: host int64 [n_texts+1], global.  h_part_offsets: host int64
 *   [n_parts+1]; part_offsets[n_parts] = n_texts.
 * h_out: host fp32 [n_texts, d_model]; row i is text i's embedding, so
 *   partition p's E_p is rows part_offsets[p] .. part_offsets[p+1]-1.
 *   h_token_ids and h_out should be pinned (hipHostMalloc); pageable memory
 *   works but its copies do not overlap.
 * copy_stream: a second stream (used only when overlap = 1); both streams
 *   may be NULL when overlap is 0 or 2.
 * h_sb_times: optional [sb_times_cap * 3] doubles; receives (upload, encode,
 *   download) ms of SuperBatch j at 3j .. 3j+2 for j < sb_times_cap.
 * stats: optional, receives the timing summary.
 * The call allocates two token and two embedding staging buffers for the
 * largest SuperBatch and frees them before returning.  Deferred device
 * errors (token IDs outside the vocabulary) are reported as by surge_check.
 */
surge_status surge_encode_all_streamed(surge_encoder* enc, int64_t n_texts,
                                       const int32_t* h_token_ids, const int64_t* h_cu_seqlens,
                                       const int64_t* h_part_offsets, int32_t n_parts,
                                       int64_t b_min, int64_t n_max, int32_t policy, float* h_out,
                                       int32_t overlap, void* compute_stream, void* copy_stream,
                                       double* h_sb_times, int64_t sb_times_cap,
                                       surge_stream_stats* stats);

/* Synchronise `hip_stream` and the encoder's last enqueued call, then report
 * deferred device-side errors (a token ID outside the vocabulary ->
 * SURGE_ERR_INVALID_ARGUMENT) and clear them. */
surge_status surge_check(surge_encoder* enc, void* hip_stream);

/*
 * Per-kernel timing with HIP events recorded on the encoder's launch stream
 * around each launch.  surge_profile_enable(enc, 1) starts recording around
 * every launch (and clears earlier records), surge_profile_enable(enc, 0)
 * stops; surge_profile_select(enc, mask) records only around the launches
 * of the kernel classes whose bit (1 << SURGE_KERNEL_*) is set in `mask`
 * (0 stops; a bit at or above SURGE_KERNEL_COUNT is an invalid argument),
 * so that timing one class adds no events between the other launches.
 * surge_profile_read synchronises on the recorded events and returns one
 * entry per kernel class (zero launches for classes not selected).
 */
#define SURGE_KERNEL_EMBED 0   /* embedding gather + LayerNorm */
#define SURGE_KERNEL_QKV 1     /* QKV projection + bias */
#define SURGE_KERNEL_ATTN 2    /* packed varlen self-attention */
#define SURGE_KERNEL_OPROJ 3   /* output projection + bias + residual */
#define SURGE_KERNEL_LN1 4     /* LayerNorm after attention */
#define SURGE_KERNEL_FFN1 5    /* FFN up-projection + bias + GELU */
#define SURGE_KERNEL_FFN2 6    /* FFN down-projection + bias + residual */
#define SURGE_KERNEL_LN2 7     /* LayerNorm after the FFN */
#define SURGE_KERNEL_POOL 8    /* mean pool + L2 + partition scatter */
#define SURGE_KERNEL_COUNT 9

typedef struct surge_kernel_stat {
  int64_t launches;
  double total_ms;  /* sum of event-measured launch durations */
  double flops;     /* algorithmic FLOPs of all launches */
  double bytes;     /* algorithmic HBM bytes of all launches */
} surge_kernel_stat;

surge_status surge_profile_enable(surge_encoder* enc, int32_t on);
surge_status surge_profile_select(surge_encoder* enc, uint32_t mask);
surge_status surge_profile_read(surge_encoder* enc, surge_kernel_stat* stats, int32_t n_stats);

#ifdef __cplusplus
}
#endif

#endif /* SURGE_H_ */
