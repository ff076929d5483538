// Host-only parts of the library: error reporting, SuperBatch formation
// (Alg. 1) and argument validation.  No HIP calls here, so everything in
// this file works without a GPU.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "internal.h"

namespace surge {

static thread_local char g_last_error[512] = "";

surge_status fail(surge_status code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return code;
}

void clear_error() { g_last_error[0] = '\0'; }

uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u);  // quiet NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

surge_status validate_desc(const surge_encoder_desc* d) {
  if (!d) return fail(SURGE_ERR_INVALID_ARGUMENT, "desc is NULL");
  if (d->n_layers < 1 || d->n_layers > 256)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "n_layers=%d outside [1, 256]", d->n_layers);
  if (d->d_model < 128 || d->d_model > 1024 || d->d_model % 128)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "d_model=%d must be a multiple of 128 in [128, 1024]",
                d->d_model);
  if (d->n_heads < 1 || d->d_model % d->n_heads)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "n_heads=%d must divide d_model=%d", d->n_heads,
                d->d_model);
  int dh = d->d_model / d->n_heads;
  if (dh != 32 && dh != 64)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "d_model/n_heads=%d must be 32 or 64", dh);
  if (d->d_ff < 128 || d->d_ff > 16384 || d->d_ff % 128)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "d_ff=%d must be a multiple of 128 in [128, 16384]",
                d->d_ff);
  if (d->vocab_size < 1) return fail(SURGE_ERR_INVALID_ARGUMENT, "vocab_size=%d", d->vocab_size);
  if (d->max_positions < 1 || d->max_positions > 4096)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "max_positions=%d outside [1, 4096]",
                d->max_positions);
  if (!(d->ln_eps >= 0.0f) || !isfinite(d->ln_eps))
    return fail(SURGE_ERR_INVALID_ARGUMENT, "ln_eps must be finite and >= 0");
  if (d->weight_dtype != SURGE_WEIGHTS_F32 && d->weight_dtype != SURGE_WEIGHTS_BF16)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "weight_dtype=%d is neither F32 (0) nor BF16 (1)",
                d->weight_dtype);
  return SURGE_OK;
}

// Alg. 1 over CSR partitions.  The aggregator holds the buffered segments and
// the running total; Flush emits one SuperBatch for a non-empty buffer.
namespace {
struct Aggregator {
  std::vector<PlanSeg> buffer;
  int64_t total = 0;
  int64_t n_sbs = 0, n_segs = 0;
  void (*emit_sb)(void*, const PlanSB&);
  void (*emit_seg)(void*, const PlanSeg&);
  void* ctx;

  void append(const PlanSeg& s) {
    buffer.push_back(s);
    total += s.count;
  }
  void flush() {
    if (buffer.empty()) return;
    PlanSB sb;
    sb.text_begin = buffer.front().first_text;
    sb.text_end = buffer.back().first_text + buffer.back().count;
    sb.seg_begin = n_segs;
    for (const PlanSeg& s : buffer) {
      if (emit_seg) emit_seg(ctx, s);
      ++n_segs;
    }
    sb.seg_end = n_segs;
    if (emit_sb) emit_sb(ctx, sb);
    ++n_sbs;
    buffer.clear();
    total = 0;
  }
};
}  // namespace

surge_status plan_superbatches(const int64_t* part_offsets, int32_t n_parts, int64_t b_min,
                               int64_t n_max, int32_t policy, void (*emit_sb)(void*, const PlanSB&),
                               void (*emit_seg)(void*, const PlanSeg&), void* ctx,
                               int64_t* n_sbs, int64_t* n_segs) {
  if (!part_offsets) return fail(SURGE_ERR_INVALID_ARGUMENT, "part_offsets is NULL");
  if (n_parts < 0) return fail(SURGE_ERR_INVALID_ARGUMENT, "n_parts=%d < 0", n_parts);
  if (b_min < 1) return fail(SURGE_ERR_INVALID_ARGUMENT, "b_min=%lld < 1", (long long)b_min);
  if (policy != SURGE_POLICY_SPLIT && policy != SURGE_POLICY_LITERAL)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "unknown policy %d", policy);
  if (part_offsets[0] != 0) return fail(SURGE_ERR_INVALID_ARGUMENT, "part_offsets[0] != 0");
  for (int32_t p = 0; p < n_parts; ++p)
    if (part_offsets[p + 1] < part_offsets[p])
      return fail(SURGE_ERR_INVALID_ARGUMENT, "part_offsets decreases at partition %d", p);
  const int64_t cap = n_max > 0 ? n_max : 0;
  Aggregator agg;
  agg.emit_sb = emit_sb;
  agg.emit_seg = emit_seg;
  agg.ctx = ctx;
  for (int32_t p = 0; p < n_parts; ++p) {
    const int64_t start = part_offsets[p];
    const int64_t n = part_offsets[p + 1] - start;
    if (n == 0) continue;  // an empty partition never reaches AddPartition
    if (policy == SURGE_POLICY_LITERAL) {
      agg.append(PlanSeg{start, n, 0, p});
      if (cap > 0 && agg.total >= cap)
        agg.flush();  // memory-safety trigger
      else if (agg.total >= b_min)
        agg.flush();  // efficiency trigger
    } else {
      if (cap > 0 && agg.total > 0 && agg.total + n > cap) agg.flush();  // pre-append safety flush
      int64_t row = 0;
      while (cap > 0 && n - row > cap) {  // oversized partition: cap-sized pieces
        agg.append(PlanSeg{start + row, cap, row, p});
        agg.flush();
        row += cap;
      }
      agg.append(PlanSeg{start + row, n - row, row, p});
      if (agg.total >= b_min) agg.flush();
    }
  }
  agg.flush();  // final Flush at the end of the stream
  if (n_sbs) *n_sbs = agg.n_sbs;
  if (n_segs) *n_segs = agg.n_segs;
  return SURGE_OK;
}

}  // namespace surge

using namespace surge;

extern "C" {

const char* surge_version(void) { return "0.1.0"; }

const char* surge_last_error(void) { return g_last_error; }

namespace {
struct PlanOut {
  surge_superbatch* sbs;
  surge_segment* segs;
  int64_t i_sb = 0, i_seg = 0;
};
void out_sb(void* c, const PlanSB& s) {
  PlanOut* o = (PlanOut*)c;
  surge_superbatch& d = o->sbs[o->i_sb++];
  d.text_begin = s.text_begin;
  d.text_end = s.text_end;
  d.seg_begin = s.seg_begin;
  d.seg_end = s.seg_end;
}
void out_seg(void* c, const PlanSeg& s) {
  PlanOut* o = (PlanOut*)c;
  surge_segment& d = o->segs[o->i_seg++];
  d.first_text = s.first_text;
  d.count = s.count;
  d.row_offset = s.row_offset;
  d.partition = s.partition;
  d.reserved = 0;
}
}  // namespace

surge_status surge_plan(const int64_t* part_offsets, int32_t n_parts, int64_t b_min, int64_t n_max,
                        int32_t policy, surge_superbatch* sbs, int64_t sb_cap, int64_t* n_sbs,
                        surge_segment* segs, int64_t seg_cap, int64_t* n_segs) {
  clear_error();
  if (!n_sbs || !n_segs) return fail(SURGE_ERR_INVALID_ARGUMENT, "n_sbs and n_segs must be set");
  int64_t ns = 0, ng = 0;
  surge_status st = plan_superbatches(part_offsets, n_parts, b_min, n_max, policy, nullptr,
                                      nullptr, nullptr, &ns, &ng);
  if (st != SURGE_OK) return st;
  *n_sbs = ns;
  *n_segs = ng;
  if (!sbs && !segs) return SURGE_OK;
  if (!sbs || !segs) return fail(SURGE_ERR_INVALID_ARGUMENT, "sbs and segs must both be set");
  if (sb_cap < ns || seg_cap < ng)
    return fail(SURGE_ERR_CAPACITY, "plan needs %lld superbatches and %lld segments",
                (long long)ns, (long long)ng);
  PlanOut o{sbs, segs};
  return plan_superbatches(part_offsets, n_parts, b_min, n_max, policy, out_sb, out_seg, &o,
                           &ns, &ng);
}

surge_status surge_validate_superbatch(const surge_encoder_desc* desc, int64_t n_texts,
                                       int64_t n_tokens, const int64_t* cu,
                                       const surge_segment* segs, int64_t n_segs,
                                       const int64_t* part_sizes, float* const* part_out,
                                       int32_t n_parts) {
  clear_error();
  surge_status st = validate_desc(desc);
  if (st != SURGE_OK) return st;
  if (n_texts < 0) return fail(SURGE_ERR_INVALID_ARGUMENT, "n_texts=%lld < 0", (long long)n_texts);
  if (n_tokens < 0 || n_tokens > (int64_t)INT32_MAX)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "n_tokens=%lld outside [0, 2^31)", (long long)n_tokens);
  if (!cu) return fail(SURGE_ERR_INVALID_ARGUMENT, "cu_seqlens is NULL");
  if (cu[0] != 0) return fail(SURGE_ERR_INVALID_ARGUMENT, "cu_seqlens[0]=%lld != 0", (long long)cu[0]);
  for (int64_t i = 0; i < n_texts; ++i) {
    int64_t L = cu[i + 1] - cu[i];
    if (L < 1 || L > desc->max_positions)
      return fail(SURGE_ERR_INVALID_ARGUMENT, "text %lld has length %lld outside [1, %d]",
                  (long long)i, (long long)L, desc->max_positions);
  }
  if (cu[n_texts] != n_tokens)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "cu_seqlens[n_texts]=%lld != n_tokens=%lld",
                (long long)cu[n_texts], (long long)n_tokens);
  if (n_segs < 0) return fail(SURGE_ERR_INVALID_ARGUMENT, "n_segs < 0");
  if (n_segs > 0 && !segs) return fail(SURGE_ERR_INVALID_ARGUMENT, "segments is NULL");
  if (n_parts < 0) return fail(SURGE_ERR_INVALID_ARGUMENT, "n_parts < 0");
  if (n_segs > 0 && (!part_sizes || !part_out))
    return fail(SURGE_ERR_INVALID_ARGUMENT, "part_sizes / part_out is NULL");
  int64_t t = 0;
  for (int64_t s = 0; s < n_segs; ++s) {
    const surge_segment& g = segs[s];
    if (g.first_text != t)
      return fail(SURGE_ERR_INVALID_ARGUMENT, "segment %lld starts at text %lld, expected %lld",
                  (long long)s, (long long)g.first_text, (long long)t);
    if (g.count < 1)
      return fail(SURGE_ERR_INVALID_ARGUMENT, "segment %lld has count %lld", (long long)s,
                  (long long)g.count);
    if (g.partition < 0 || g.partition >= n_parts)
      return fail(SURGE_ERR_INVALID_ARGUMENT, "segment %lld names partition %d outside [0, %d)",
                  (long long)s, g.partition, n_parts);
    if (g.row_offset < 0 || g.row_offset + g.count > part_sizes[g.partition])
      return fail(SURGE_ERR_INVALID_ARGUMENT,
                  "segment %lld rows [%lld, %lld) overflow partition %d of %lld rows", (long long)s,
                  (long long)g.row_offset, (long long)(g.row_offset + g.count), g.partition,
                  (long long)part_sizes[g.partition]);
    if (!part_out[g.partition])
      return fail(SURGE_ERR_INVALID_ARGUMENT, "output of partition %d is NULL", g.partition);
    t += g.count;
  }
  if (t != n_texts)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "segments cover %lld texts, expected %lld", (long long)t,
                (long long)n_texts);
  return SURGE_OK;
}

surge_status surge_validate_input(const surge_encoder_desc* desc, int64_t n_texts,
                                  const int64_t* cu, const int64_t* part_offsets, int32_t n_parts,
                                  int64_t b_min, int64_t n_max, int32_t policy,
                                  float* const* part_out, int64_t* n_superbatches,
                                  int64_t* max_sb_texts, int64_t* max_sb_tokens) {
  clear_error();
  surge_status st = validate_desc(desc);
  if (st != SURGE_OK) return st;
  if (!cu || !part_offsets) return fail(SURGE_ERR_INVALID_ARGUMENT, "NULL host array");
  if (n_texts < 0) return fail(SURGE_ERR_INVALID_ARGUMENT, "n_texts=%lld < 0", (long long)n_texts);
  if (n_parts < 0) return fail(SURGE_ERR_INVALID_ARGUMENT, "n_parts=%d < 0", n_parts);
  if (part_offsets[n_parts] != n_texts)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "part_offsets[n_parts]=%lld != n_texts=%lld",
                (long long)part_offsets[n_parts], (long long)n_texts);
  if (cu[0] != 0) return fail(SURGE_ERR_INVALID_ARGUMENT, "cu_seqlens[0]=%lld != 0", (long long)cu[0]);
  for (int64_t i = 0; i < n_texts; ++i) {
    const int64_t L = cu[i + 1] - cu[i];
    if (L < 1 || L > desc->max_positions)
      return fail(SURGE_ERR_INVALID_ARGUMENT, "text %lld has length %lld outside [1, %d]",
                  (long long)i, (long long)L, desc->max_positions);
  }
  // The plan (this also checks part_offsets, b_min and the policy).
  struct Scan {
    const int64_t* cu;
    int64_t n = 0, max_texts = 0, max_tokens = 0;
  } scan{cu};
  auto on_sb = [](void* c, const PlanSB& s) {
    Scan* q = (Scan*)c;
    ++q->n;
    q->max_texts = std::max(q->max_texts, s.text_end - s.text_begin);
    q->max_tokens = std::max(q->max_tokens, q->cu[s.text_end] - q->cu[s.text_begin]);
  };
  int64_t ns = 0, ng = 0;
  st = plan_superbatches(part_offsets, n_parts, b_min, n_max, policy, on_sb, nullptr, &scan, &ns,
                         &ng);
  if (st != SURGE_OK) return st;
  if (scan.max_tokens > (int64_t)INT32_MAX)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "a SuperBatch holds %lld tokens (>= 2^31)",
                (long long)scan.max_tokens);
  if (n_texts > 0 && !part_out) return fail(SURGE_ERR_INVALID_ARGUMENT, "part_out is NULL");
  for (int32_t p = 0; p < n_parts; ++p)
    if (part_offsets[p + 1] > part_offsets[p] && !part_out[p])
      return fail(SURGE_ERR_INVALID_ARGUMENT, "output of partition %d is NULL", p);
  if (n_superbatches) *n_superbatches = ns;
  if (max_sb_texts) *max_sb_texts = scan.max_texts;
  if (max_sb_tokens) *max_sb_tokens = scan.max_tokens;
  return SURGE_OK;
}

}  // extern "C"
