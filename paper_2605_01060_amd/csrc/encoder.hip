// The encoder object and the SuperBatch encode path.
//
// Create: validate the description, round matrices and embedding tables to
// bf16, transpose every matrix to [out, in] (K-contiguous for the MFMA
// linear kernel) and upload everything in one device block; allocate the
// activation workspace for max_tokens_per_chunk tokens.
//
// Encode one SuperBatch (Alg. 1, Flush): validate on the host, resolve every
// text's output row pointer from the segment table, cut the SuperBatch into
// token chunks at text boundaries, and for each chunk upload (cu_seqlens,
// row pointers) through a pinned staging ring and launch
//   embed+LN, then per layer: QKV, attention, O-proj+residual, LN1,
//   FFN1+GELU, FFN2+residual, LN2, and finally pool+L2+scatter.
// Everything is enqueued on the caller's stream; nothing blocks except the
// reuse of a staging slot whose previous copy is still pending.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "internal.h"
#include "kernels.h"

using namespace surge;

namespace {

constexpr int kStagingSlots = 4;

struct LayerWeights {
  uint16_t *wqkv, *wo, *w1, *w2;               // bf16 [out, in]
  float *bqkv, *bo, *ln1g, *ln1b, *b1, *b2, *ln2g, *ln2b;  // fp32
  // The LayerNorm before the QKV (layers >= 1: the previous layer's LN2) and
  // before FFN1 (LN1) is folded into those GEMMs: W' = W diag(gamma) is what
  // wqkv / w1 hold, s = row sums of W', and bqkv / b1 hold b + W beta.
  float *sqkv, *s1;                            // fp32 [3d], [d_ff]
};

struct ProfRecord {
  int kind;
  int ev;  // index of the start event; stop is ev + 1
  double flops, bytes;
};

}  // namespace

struct surge_encoder {
  surge_encoder_desc desc;
  int device = 0;
  int64_t max_tokens = 0;
  // weights
  void* wblock = nullptr;
  uint16_t *word = nullptr, *pos = nullptr;
  float *lneg = nullptr, *lneb = nullptr;
  std::vector<LayerWeights> layers;
  // workspace
  void* wsblock = nullptr;
  int64_t ws_bytes = 0;
  uint16_t *X = nullptr, *QKV = nullptr, *CTX = nullptr, *Y = nullptr, *H = nullptr;
  float2 *SX = nullptr, *SY = nullptr;  // row statistics partials of X and Y
  float2 *RX = nullptr, *RY = nullptr;  // their per-row LayerNorm factors
  int32_t* d_cu = nullptr;     // [max_tokens + 1]
  uint64_t* d_dst = nullptr;   // [max_tokens]
  uint32_t* d_items = nullptr; // [max_tokens] attention work items
  int* d_err = nullptr;
  int n_cus = 0;  // compute units of the device (GEMM grid size)
  // The workspace is shared by every call: each call's stream waits for the
  // previous call's last work, which this event marks.
  hipEvent_t last_use = nullptr;
  bool last_use_recorded = false;
  // pinned staging ring for chunk metadata
  void* staging[kStagingSlots] = {};
  hipEvent_t staging_ev[kStagingSlots] = {};
  bool staging_used[kStagingSlots] = {};
  int staging_next = 0;
  size_t staging_bytes = 0;
  // host scratch
  std::vector<uint64_t> h_dst;
  std::vector<int64_t> h_lcu;
  // profiling
  uint32_t prof_kinds = 0;  // bit k set: time launches of kernel class k
  std::vector<hipEvent_t> prof_events;
  int prof_used = 0;
  std::vector<ProfRecord> prof_recs;
};

#define HIP_TRY(expr)                                                                    \
  do {                                                                                   \
    hipError_t e_ = (expr);                                                              \
    if (e_ != hipSuccess)                                                                \
      return fail(e_ == hipErrorOutOfMemory ? SURGE_ERR_OUT_OF_MEMORY : SURGE_ERR_DEVICE, \
                  "%s failed: %s", #expr, hipGetErrorString(e_));                        \
  } while (0)

namespace {

void free_encoder(surge_encoder* e) {
  if (!e) return;
  hipSetDevice(e->device);
  hipDeviceSynchronize();
  for (int i = 0; i < kStagingSlots; ++i) {
    if (e->staging_ev[i]) hipEventDestroy(e->staging_ev[i]);
    if (e->staging[i]) hipHostFree(e->staging[i]);
  }
  for (hipEvent_t ev : e->prof_events) hipEventDestroy(ev);
  if (e->last_use) hipEventDestroy(e->last_use);
  if (e->wblock) hipFree(e->wblock);
  if (e->wsblock) hipFree(e->wsblock);
  delete e;
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Profiling: start/stop event pair around one launch of a selected class.
surge_status prof_begin(surge_encoder* e, hipStream_t s, int kind, int* ev) {
  if (!((e->prof_kinds >> kind) & 1u)) return SURGE_OK;
  if ((size_t)e->prof_used + 2 > e->prof_events.size()) {
    for (int i = 0; i < 256; ++i) {
      hipEvent_t x;
      HIP_TRY(hipEventCreate(&x));
      e->prof_events.push_back(x);
    }
  }
  *ev = e->prof_used;
  e->prof_used += 2;
  HIP_TRY(hipEventRecord(e->prof_events[*ev], s));
  return SURGE_OK;
}

surge_status prof_end(surge_encoder* e, hipStream_t s, int ev, int kind, double flops,
                      double bytes) {
  if (ev < 0) return SURGE_OK;
  HIP_TRY(hipEventRecord(e->prof_events[ev + 1], s));
  e->prof_recs.push_back(ProfRecord{kind, ev, flops, bytes});
  return SURGE_OK;
}

#define LAUNCH(kind, flops, bytes, call)                             \
  do {                                                               \
    int ev_ = -1;                                                    \
    surge_status st_ = prof_begin(e, stream, kind, &ev_);            \
    if (st_ != SURGE_OK) return st_;                                 \
    hipError_t le_ = (call);                                         \
    if (le_ != hipSuccess)                                           \
      return fail(SURGE_ERR_DEVICE, "kernel launch failed: %s", hipGetErrorString(le_)); \
    st_ = prof_end(e, stream, ev_, kind, flops, bytes);              \
    if (st_ != SURGE_OK) return st_;                                 \
  } while (0)

// Order a call after the encoder's previous one: `stream` waits for the
// event recorded at the end of that call (a no-op before the first call).
surge_status begin_call(surge_encoder* e, hipStream_t stream) {
  if (e->last_use_recorded) HIP_TRY(hipStreamWaitEvent(stream, e->last_use, 0));
  return SURGE_OK;
}

surge_status end_call(surge_encoder* e, hipStream_t stream) {
  HIP_TRY(hipEventRecord(e->last_use, stream));
  e->last_use_recorded = true;
  return SURGE_OK;
}

// Encode texts [0, n_texts) of a validated SuperBatch whose row pointers are
// in e->h_dst.  cu is SuperBatch-local host int64.
surge_status encode_chunks(surge_encoder* e, int64_t n_texts, const int32_t* d_tokens,
                           const int64_t* cu, hipStream_t stream) {
  const surge_encoder_desc& D = e->desc;
  const int d = D.d_model, f = D.d_ff, dh = d / D.n_heads;
  int64_t t0 = 0;
  while (t0 < n_texts) {
    // Largest run of whole texts that fits the workspace.
    int64_t t1 = t0;
    while (t1 < n_texts && cu[t1 + 1] - cu[t0] <= e->max_tokens) ++t1;
    const int64_t S = t1 - t0;
    const int64_t T = cu[t1] - cu[t0];

    // Stage (cu32 [S+1], dst [S], attention items) in a pinned slot, then
    // copy to the device.
    const int slot = e->staging_next;
    e->staging_next = (slot + 1) % kStagingSlots;
    if (e->staging_used[slot]) HIP_TRY(hipEventSynchronize(e->staging_ev[slot]));
    char* stg = (char*)e->staging[slot];
    const size_t cu_region = align_up((size_t)(e->max_tokens + 1) * 4, 16);
    const size_t dst_region = (size_t)e->max_tokens * 8;
    int32_t* hcu = (int32_t*)stg;
    uint64_t* hdst = (uint64_t*)(stg + cu_region);
    uint32_t* hitems = (uint32_t*)(stg + cu_region + dst_region);
    for (int64_t i = 0; i <= S; ++i) hcu[i] = (int32_t)(cu[t0 + i] - cu[t0]);
    memcpy(hdst, e->h_dst.data() + t0, (size_t)S * 8);
    e->h_lcu.resize((size_t)S + 1);
    for (int64_t i = 0; i <= S; ++i) e->h_lcu[(size_t)i] = cu[t0 + i] - cu[t0];
    const int n_items = row_block_items(e->h_lcu.data(), S, hitems);
    const size_t cu_bytes = align_up((size_t)(S + 1) * 4, 16);
    HIP_TRY(hipMemcpyAsync(e->d_cu, hcu, cu_bytes, hipMemcpyHostToDevice, stream));
    HIP_TRY(hipMemcpyAsync(e->d_dst, hdst, (size_t)S * 8, hipMemcpyHostToDevice, stream));
    HIP_TRY(hipMemcpyAsync(e->d_items, hitems, (size_t)n_items * 4, hipMemcpyHostToDevice, stream));
    HIP_TRY(hipEventRecord(e->staging_ev[slot], stream));
    e->staging_used[slot] = true;

    const int32_t* toks = d_tokens + cu[t0];
    double sumL2 = 0.0;
    for (int64_t i = t0; i < t1; ++i) {
      const double L = (double)(cu[i + 1] - cu[i]);
      sumL2 += L * L;
    }
    const double Td = (double)T;
    const int Si = (int)S;

    LAUNCH(SURGE_KERNEL_EMBED, 0.0, Td * (4.0 + 6.0 * d),
           launch_embed_ln(toks, e->d_cu, e->d_items, n_items, e->word, e->pos, e->lneg,
                           e->lneb, D.ln_eps, D.vocab_size, d, e->X, e->d_err, stream));
    // Post-LN with the LayerNorms folded into their neighbours: X and Y
    // hold raw (pre-LN) residual rows, SX and SY their statistics partials
    // (written by the residual GEMMs), RX and RY the per-row factors.
    const int parts = d / linear_stats_width(T, d);  // partials of a [T, d] output
    for (int l = 0; l < D.n_layers; ++l) {
      const LayerWeights& w = e->layers[l];
      const LayerWeights* pw = l > 0 ? &e->layers[l - 1] : nullptr;
      LinearExtra xq;  // QKV: LN2 of the previous layer folded in (layer 0: plain)
      xq.n_cus = e->n_cus;
      xq.rows_in = e->RX;
      xq.col_s = w.sqkv;
      LAUNCH(SURGE_KERNEL_QKV, 2.0 * Td * d * 3 * d, 2.0 * (Td * d + 3.0 * d * d + Td * 3 * d),
             launch_linear(e->X, w.wqkv, w.bqkv, nullptr, e->QKV, T, 3 * d, d,
                           l == 0 ? EPI_BIAS : EPI_FOLD, xq, stream));
      LAUNCH(SURGE_KERNEL_ATTN, 4.0 * d * sumL2, 2.0 * Td * 4 * d,
             launch_attention(e->QKV, e->CTX, e->d_cu, e->d_items, n_items, D.n_heads, dh, stream));
      LinearExtra xo;  // O-proj + residual (LN2 of the previous layer applied to it)
      xo.n_cus = e->n_cus;
      xo.rows_in = e->RX;
      xo.stats_out = e->SY;
      xo.gamma = pw ? pw->ln2g : nullptr;
      xo.beta = pw ? pw->ln2b : nullptr;
      LAUNCH(SURGE_KERNEL_OPROJ, 2.0 * Td * d * d, 2.0 * (3.0 * Td * d + (double)d * d),
             launch_linear(e->CTX, w.wo, w.bo, e->X, e->Y, T, d, d,
                           l == 0 ? EPI_RES_STATS : EPI_LNRES_STATS, xo, stream));
      LAUNCH(SURGE_KERNEL_LN1, 0.0, Td * (8.0 * parts + 8.0),
             launch_ln_rows(e->SY, parts, T, D.ln_eps, e->RY, stream));
      LinearExtra x1;  // FFN1: LN1 folded in
      x1.n_cus = e->n_cus;
      x1.rows_in = e->RY;
      x1.col_s = w.s1;
      LAUNCH(SURGE_KERNEL_FFN1, 2.0 * Td * d * f, 2.0 * (Td * d + (double)d * f + Td * f),
             launch_linear(e->Y, w.w1, w.b1, nullptr, e->H, T, f, d, EPI_FOLD_GELU, x1, stream));
      LinearExtra x2;  // FFN2 + residual LN1(Y)
      x2.n_cus = e->n_cus;
      x2.rows_in = e->RY;
      x2.stats_out = e->SX;
      x2.gamma = w.ln1g;
      x2.beta = w.ln1b;
      LAUNCH(SURGE_KERNEL_FFN2, 2.0 * Td * d * f, 2.0 * (Td * f + (double)d * f + 2.0 * Td * d),
             launch_linear(e->H, w.w2, w.b2, e->Y, e->X, T, d, f, EPI_LNRES_STATS, x2, stream));
      LAUNCH(SURGE_KERNEL_LN2, 0.0, Td * (8.0 * parts + 8.0),
             launch_ln_rows(e->SX, parts, T, D.ln_eps, e->RX, stream));
    }
    // The last layer's LN2 is applied inside the pooling.
    const LayerWeights& wl = e->layers[D.n_layers - 1];
    LAUNCH(SURGE_KERNEL_POOL, 0.0, 2.0 * Td * d + 8.0 * Td + 4.0 * S * d,
           launch_pool_l2_scatter(e->X, e->d_cu, Si, e->d_dst, d, e->RX, wl.ln2g, wl.ln2b,
                                  stream));
    t0 = t1;
  }
  return SURGE_OK;
}

// Resolve text -> output row pointer from a validated segment table.
void resolve_rows(surge_encoder* e, int64_t n_texts, const surge_segment* segs, int64_t n_segs,
                  float* const* part_out) {
  e->h_dst.resize((size_t)n_texts);
  const int64_t d = e->desc.d_model;
  for (int64_t s = 0; s < n_segs; ++s) {
    const surge_segment& g = segs[s];
    float* base = part_out[g.partition] + g.row_offset * d;
    for (int64_t k = 0; k < g.count; ++k)
      e->h_dst[(size_t)(g.first_text + k)] = (uint64_t)(uintptr_t)(base + k * d);
  }
}

surge_status check_alignment(int64_t n_segs, const surge_segment* segs, float* const* part_out) {
  for (int64_t s = 0; s < n_segs; ++s)
    if (((uintptr_t)part_out[segs[s].partition]) & 15u)
      return fail(SURGE_ERR_INVALID_ARGUMENT, "output of partition %d is not 16-byte aligned",
                  segs[s].partition);
  return SURGE_OK;
}

// The SuperBatches of a whole input and their segments (global text
// indices), from the host planner.
struct Plan {
  std::vector<PlanSB> sbs;
  std::vector<surge_segment> segs;
};

surge_status make_plan(const int64_t* part_offsets, int32_t n_parts, int64_t b_min, int64_t n_max,
                       int32_t policy, Plan* plan, int64_t* n_sbs) {
  auto on_sb = [](void* c, const PlanSB& s) { ((Plan*)c)->sbs.push_back(s); };
  auto on_seg = [](void* c, const PlanSeg& s) {
    surge_segment g;
    g.first_text = s.first_text;
    g.count = s.count;
    g.row_offset = s.row_offset;
    g.partition = s.partition;
    g.reserved = 0;
    ((Plan*)c)->segs.push_back(g);
  };
  int64_t ng = 0;
  return plan_superbatches(part_offsets, n_parts, b_min, n_max, policy, on_sb, on_seg, plan, n_sbs,
                           &ng);
}

}  // namespace

extern "C" {

surge_status surge_encoder_create(const surge_encoder_desc* desc, const void* const* host_weights_in,
                                  int32_t n_weights, int64_t max_tokens_per_chunk,
                                  surge_encoder** out) {
  clear_error();
  if (!out) return fail(SURGE_ERR_INVALID_ARGUMENT, "out is NULL");
  *out = nullptr;
  surge_status st = validate_desc(desc);
  if (st != SURGE_OK) return st;
  const surge_encoder_desc D = *desc;
  const int64_t expect = 4 + 12 * (int64_t)D.n_layers;
  if (!host_weights_in || n_weights != expect)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "expected %lld weight arrays, got %d",
                (long long)expect, n_weights);
  for (int i = 0; i < n_weights; ++i)
    if (!host_weights_in[i]) return fail(SURGE_ERR_INVALID_ARGUMENT, "weight %d is NULL", i);
  if (max_tokens_per_chunk < D.max_positions || max_tokens_per_chunk > (int64_t)1 << 25)
    return fail(SURGE_ERR_INVALID_ARGUMENT,
                "max_tokens_per_chunk=%lld outside [max_positions, 2^25]",
                (long long)max_tokens_per_chunk);

  surge_encoder* e = new surge_encoder();
  e->desc = D;
  e->max_tokens = max_tokens_per_chunk;
  hipError_t he = hipGetDevice(&e->device);
  if (he != hipSuccess) {
    delete e;
    return fail(SURGE_ERR_DEVICE, "hipGetDevice failed: %s", hipGetErrorString(he));
  }

  const int64_t d = D.d_model, f = D.d_ff, V = D.vocab_size, P = D.max_positions;
  // Element counts of the weight arrays, in the fixed order.
  std::vector<int64_t> counts = {V * d, P * d, d, d};
  for (int l = 0; l < D.n_layers; ++l) {
    const int64_t per[12] = {d * 3 * d, 3 * d, d * d, d, d, d, d * f, f, f * d, d, d, d};
    counts.insert(counts.end(), per, per + 12);
  }
  // bf16 input: every array widened exactly to float32 first, so both input
  // types go through the same rounding and folding below.
  std::vector<std::vector<float>> widened;
  std::vector<const float*> hw((size_t)n_weights);
  if (D.weight_dtype == SURGE_WEIGHTS_BF16) {
    widened.resize((size_t)n_weights);
    for (int i = 0; i < n_weights; ++i) {
      const uint16_t* src = (const uint16_t*)host_weights_in[i];
      std::vector<float>& dst = widened[(size_t)i];
      dst.resize((size_t)counts[(size_t)i]);
      for (int64_t k = 0; k < counts[(size_t)i]; ++k) {
        const uint32_t bits = (uint32_t)src[k] << 16;
        memcpy(&dst[(size_t)k], &bits, 4);
      }
      hw[(size_t)i] = dst.data();
    }
  } else {
    for (int i = 0; i < n_weights; ++i) hw[(size_t)i] = (const float*)host_weights_in[i];
  }
  const float* const* host_weights = hw.data();
  // Device weight block layout (byte offsets, 256-aligned pieces).
  std::vector<size_t> offs;
  size_t total = 0;
  auto take = [&](size_t bytes) {
    size_t o = total;
    total = align_up(total + bytes, 256);
    offs.push_back(o);
    return o;
  };
  take((size_t)V * d * 2);  // word
  take((size_t)P * d * 2);  // pos
  take((size_t)d * 4);      // ln_e gamma
  take((size_t)d * 4);      // ln_e beta
  const int64_t mshape[4][2] = {{d, 3 * d}, {d, d}, {d, f}, {f, d}};  // [in, out]
  for (int l = 0; l < D.n_layers; ++l) {
    take((size_t)d * 3 * d * 2);  // wqkv
    take((size_t)3 * d * 4);      // bqkv
    take((size_t)d * d * 2);      // wo
    take((size_t)d * 4);          // bo
    take((size_t)d * 4);          // ln1g
    take((size_t)d * 4);          // ln1b
    take((size_t)d * f * 2);      // w1
    take((size_t)f * 4);          // b1
    take((size_t)f * d * 2);      // w2
    take((size_t)d * 4);          // b2
    take((size_t)d * 4);          // ln2g
    take((size_t)d * 4);          // ln2b
  }
  const size_t extra0 = offs.size();  // per layer: sqkv, s1
  for (int l = 0; l < D.n_layers; ++l) {
    take((size_t)3 * d * 4);
    take((size_t)f * 4);
  }
  (void)mshape;
  std::vector<uint8_t> host(total, 0);
  auto put_bf16 = [&](int idx, const float* src, int64_t n) {
    uint16_t* dst = (uint16_t*)(host.data() + offs[idx]);
    for (int64_t i = 0; i < n; ++i) dst[i] = f32_to_bf16_rne(src[i]);
  };
  auto put_bf16_t = [&](int idx, const float* src, int64_t in, int64_t outn) {
    // src [in, out] row-major -> dst [out, in]
    uint16_t* dst = (uint16_t*)(host.data() + offs[idx]);
    for (int64_t i = 0; i < in; ++i)
      for (int64_t o = 0; o < outn; ++o) dst[o * in + i] = f32_to_bf16_rne(src[i * outn + o]);
  };
  auto put_f32 = [&](int idx, const float* src, int64_t n) {
    memcpy(host.data() + offs[idx], src, (size_t)n * 4);
  };
  // LayerNorm folding: src [in, out] row-major -> dst [out, in] holding
  // bf16(W[i][o] gamma[i]) (one rounding), s[o] = sum_i dst[o][i] (the
  // rounded values the GEMM uses), b'[o] = b[o] + sum_i W[i][o] beta[i].
  auto put_folded = [&](int widx, int bidx, size_t sidx, const float* src, const float* bias,
                        const float* gamma, const float* beta, int64_t in, int64_t outn) {
    uint16_t* dst = (uint16_t*)(host.data() + offs[widx]);
    float* bo = (float*)(host.data() + offs[bidx]);
    float* so = (float*)(host.data() + offs[sidx]);
    std::vector<double> ssum((size_t)outn, 0.0), csum((size_t)outn, 0.0);
    for (int64_t i = 0; i < in; ++i)
      for (int64_t o = 0; o < outn; ++o) {
        const float wv = src[i * outn + o];
        const uint16_t q = f32_to_bf16_rne(wv * gamma[i]);
        dst[o * in + i] = q;
        uint32_t bits = (uint32_t)q << 16;
        float qf;
        memcpy(&qf, &bits, 4);
        ssum[(size_t)o] += (double)qf;
        csum[(size_t)o] += (double)wv * (double)beta[i];
      }
    for (int64_t o = 0; o < outn; ++o) {
      so[o] = (float)ssum[(size_t)o];
      bo[o] = (float)((double)bias[o] + csum[(size_t)o]);
    }
  };
  put_bf16(0, host_weights[0], V * d);
  put_bf16(1, host_weights[1], P * d);
  put_f32(2, host_weights[2], d);
  put_f32(3, host_weights[3], d);
  for (int l = 0; l < D.n_layers; ++l) {
    const int b = 4 + 12 * l;
    if (l == 0) {  // input: the embedding LN's output, already normalised
      put_bf16_t(b + 0, host_weights[b + 0], d, 3 * d);
      put_f32(b + 1, host_weights[b + 1], 3 * d);
    } else {
      const int pb = 4 + 12 * (l - 1);  // previous layer's LN2
      put_folded(b + 0, b + 1, extra0 + 2 * l, host_weights[b + 0], host_weights[b + 1],
                 host_weights[pb + 10], host_weights[pb + 11], d, 3 * d);
    }
    put_bf16_t(b + 2, host_weights[b + 2], d, d);
    put_f32(b + 3, host_weights[b + 3], d);
    put_f32(b + 4, host_weights[b + 4], d);
    put_f32(b + 5, host_weights[b + 5], d);
    put_folded(b + 6, b + 7, extra0 + 2 * l + 1, host_weights[b + 6], host_weights[b + 7],
               host_weights[b + 4], host_weights[b + 5], d, f);
    put_bf16_t(b + 8, host_weights[b + 8], f, d);
    put_f32(b + 9, host_weights[b + 9], d);
    put_f32(b + 10, host_weights[b + 10], d);
    put_f32(b + 11, host_weights[b + 11], d);
  }

  auto cleanup_fail = [&](surge_status code) {
    free_encoder(e);
    return code;
  };
  hipError_t err = hipMalloc(&e->wblock, total);
  if (err != hipSuccess)
    return cleanup_fail(fail(SURGE_ERR_OUT_OF_MEMORY, "weights: hipMalloc(%zu) failed: %s", total,
                             hipGetErrorString(err)));
  err = hipMemcpy(e->wblock, host.data(), total, hipMemcpyHostToDevice);
  if (err != hipSuccess)
    return cleanup_fail(fail(SURGE_ERR_DEVICE, "weights: hipMemcpy failed: %s", hipGetErrorString(err)));
  char* wb = (char*)e->wblock;
  e->word = (uint16_t*)(wb + offs[0]);
  e->pos = (uint16_t*)(wb + offs[1]);
  e->lneg = (float*)(wb + offs[2]);
  e->lneb = (float*)(wb + offs[3]);
  for (int l = 0; l < D.n_layers; ++l) {
    const int b = 4 + 12 * l;
    LayerWeights w;
    w.wqkv = (uint16_t*)(wb + offs[b + 0]);
    w.bqkv = (float*)(wb + offs[b + 1]);
    w.wo = (uint16_t*)(wb + offs[b + 2]);
    w.bo = (float*)(wb + offs[b + 3]);
    w.ln1g = (float*)(wb + offs[b + 4]);
    w.ln1b = (float*)(wb + offs[b + 5]);
    w.w1 = (uint16_t*)(wb + offs[b + 6]);
    w.b1 = (float*)(wb + offs[b + 7]);
    w.w2 = (uint16_t*)(wb + offs[b + 8]);
    w.b2 = (float*)(wb + offs[b + 9]);
    w.ln2g = (float*)(wb + offs[b + 10]);
    w.ln2b = (float*)(wb + offs[b + 11]);
    w.sqkv = l == 0 ? nullptr : (float*)(wb + offs[extra0 + 2 * l]);
    w.s1 = (float*)(wb + offs[extra0 + 2 * l + 1]);
    e->layers.push_back(w);
  }

  // Workspace: X, QKV, CTX, Y, H activations + metadata + error flag.
  const int64_t T = max_tokens_per_chunk;
  size_t ws = 0;
  std::vector<size_t> wo;
  auto wtake = [&](size_t bytes) {
    size_t o = ws;
    ws = align_up(ws + bytes, 256);
    wo.push_back(o);
  };
  wtake((size_t)T * d * 2);        // X
  wtake((size_t)T * 3 * d * 2);    // QKV
  wtake((size_t)T * d * 2);        // CTX
  wtake((size_t)T * d * 2);        // Y
  wtake((size_t)T * f * 2);        // H
  wtake((size_t)(T + 1) * 4 + 16); // cu
  wtake((size_t)T * 8);            // dst
  wtake((size_t)T * 4);            // attention items
  wtake(256);                      // err
  wtake((size_t)T * (d / 64) * 8); // SX: at most d/64 partials per row
  wtake((size_t)T * (d / 64) * 8); // SY
  wtake((size_t)T * 8);            // RX
  wtake((size_t)T * 8);            // RY
  err = hipMalloc(&e->wsblock, ws);
  if (err != hipSuccess)
    return cleanup_fail(fail(SURGE_ERR_OUT_OF_MEMORY, "workspace: hipMalloc(%zu) failed: %s", ws,
                             hipGetErrorString(err)));
  e->ws_bytes = (int64_t)ws;
  char* w = (char*)e->wsblock;
  e->X = (uint16_t*)(w + wo[0]);
  e->QKV = (uint16_t*)(w + wo[1]);
  e->CTX = (uint16_t*)(w + wo[2]);
  e->Y = (uint16_t*)(w + wo[3]);
  e->H = (uint16_t*)(w + wo[4]);
  e->d_cu = (int32_t*)(w + wo[5]);
  e->d_dst = (uint64_t*)(w + wo[6]);
  e->d_items = (uint32_t*)(w + wo[7]);
  e->d_err = (int*)(w + wo[8]);
  e->SX = (float2*)(w + wo[9]);
  e->SY = (float2*)(w + wo[10]);
  e->RX = (float2*)(w + wo[11]);
  e->RY = (float2*)(w + wo[12]);
  err = hipMemset(e->d_err, 0, 256);
  if (err != hipSuccess)
    return cleanup_fail(fail(SURGE_ERR_DEVICE, "hipMemset failed: %s", hipGetErrorString(err)));

  err = hipDeviceGetAttribute(&e->n_cus, hipDeviceAttributeMultiprocessorCount, e->device);
  if (err != hipSuccess)
    return cleanup_fail(fail(SURGE_ERR_DEVICE, "hipDeviceGetAttribute failed: %s",
                             hipGetErrorString(err)));
  err = hipEventCreateWithFlags(&e->last_use, hipEventDisableTiming);
  if (err != hipSuccess)
    return cleanup_fail(fail(SURGE_ERR_DEVICE, "hipEventCreate failed: %s", hipGetErrorString(err)));

  e->staging_bytes = align_up((size_t)(T + 1) * 4, 16) + (size_t)T * 8 + (size_t)T * 4;
  for (int i = 0; i < kStagingSlots; ++i) {
    err = hipHostMalloc(&e->staging[i], e->staging_bytes, hipHostMallocDefault);
    if (err != hipSuccess)
      return cleanup_fail(fail(SURGE_ERR_OUT_OF_MEMORY, "hipHostMalloc failed: %s",
                               hipGetErrorString(err)));
    err = hipEventCreateWithFlags(&e->staging_ev[i], hipEventDisableTiming);
    if (err != hipSuccess)
      return cleanup_fail(fail(SURGE_ERR_DEVICE, "hipEventCreate failed: %s", hipGetErrorString(err)));
  }
  *out = e;
  return SURGE_OK;
}

void surge_encoder_destroy(surge_encoder* enc) { free_encoder(enc); }

surge_status surge_encoder_info(const surge_encoder* enc, surge_encoder_desc* desc,
                                int64_t* max_tokens_per_chunk, int64_t* workspace_bytes) {
  clear_error();
  if (!enc) return fail(SURGE_ERR_INVALID_ARGUMENT, "encoder is NULL");
  if (desc) *desc = enc->desc;
  if (max_tokens_per_chunk) *max_tokens_per_chunk = enc->max_tokens;
  if (workspace_bytes) *workspace_bytes = enc->ws_bytes;
  return SURGE_OK;
}

surge_status surge_encode_superbatch(surge_encoder* enc, int64_t n_texts, int64_t n_tokens,
                                     const int32_t* d_token_ids, const int64_t* h_cu_seqlens,
                                     const surge_segment* h_segs, int64_t n_segs,
                                     float* const* h_part_out, const int64_t* h_part_sizes,
                                     int32_t n_parts, void* hip_stream) {
  clear_error();
  if (!enc) return fail(SURGE_ERR_INVALID_ARGUMENT, "encoder is NULL");
  surge_status st = surge_validate_superbatch(&enc->desc, n_texts, n_tokens, h_cu_seqlens, h_segs,
                                              n_segs, h_part_sizes, h_part_out, n_parts);
  if (st != SURGE_OK) return st;
  if (n_texts > 0 && !d_token_ids) return fail(SURGE_ERR_INVALID_ARGUMENT, "token_ids is NULL");
  st = check_alignment(n_segs, h_segs, h_part_out);
  if (st != SURGE_OK) return st;
  if (n_texts == 0) return SURGE_OK;
  HIP_TRY(hipSetDevice(enc->device));
  surge_encoder* e = enc;
  const hipStream_t stream = (hipStream_t)hip_stream;
  resolve_rows(e, n_texts, h_segs, n_segs, h_part_out);
  st = begin_call(e, stream);
  if (st != SURGE_OK) return st;
  st = encode_chunks(e, n_texts, d_token_ids, h_cu_seqlens, stream);
  if (st != SURGE_OK) return st;
  return end_call(e, stream);
}

surge_status surge_encode_all(surge_encoder* enc, int64_t n_texts, const int32_t* d_token_ids,
                              const int64_t* h_cu_seqlens, const int64_t* h_part_offsets,
                              int32_t n_parts, int64_t b_min, int64_t n_max, int32_t policy,
                              float* const* h_part_out, int64_t first_sb, int64_t* n_superbatches,
                              void* hip_stream) {
  clear_error();
  if (!enc) return fail(SURGE_ERR_INVALID_ARGUMENT, "encoder is NULL");
  if (first_sb < 0) return fail(SURGE_ERR_INVALID_ARGUMENT, "first_sb < 0");
  // Validate the whole input once (int64 offsets, no cap on the total token
  // count), then every SuperBatch of the plan is consistent.
  surge_status st = surge_validate_input(&enc->desc, n_texts, h_cu_seqlens, h_part_offsets,
                                         n_parts, b_min, n_max, policy, h_part_out, nullptr,
                                         nullptr, nullptr);
  if (st != SURGE_OK) return st;
  Plan ctx;
  int64_t ns = 0;
  st = make_plan(h_part_offsets, n_parts, b_min, n_max, policy, &ctx, &ns);
  if (st != SURGE_OK) return st;
  if (n_superbatches) *n_superbatches = ns;
  st = check_alignment((int64_t)ctx.segs.size(), ctx.segs.data(), h_part_out);
  if (st != SURGE_OK) return st;
  if (n_texts > 0 && !d_token_ids) return fail(SURGE_ERR_INVALID_ARGUMENT, "token_ids is NULL");
  if (n_texts == 0) return SURGE_OK;
  HIP_TRY(hipSetDevice(enc->device));
  surge_encoder* e = enc;
  const hipStream_t stream = (hipStream_t)hip_stream;
  st = begin_call(e, stream);
  if (st != SURGE_OK) return st;
  std::vector<int64_t> lcu;
  for (int64_t k = first_sb; k < ns; ++k) {
    const PlanSB& sb = ctx.sbs[(size_t)k];
    const int64_t S = sb.text_end - sb.text_begin;
    lcu.resize((size_t)S + 1);
    const int64_t base = h_cu_seqlens[sb.text_begin];
    for (int64_t i = 0; i <= S; ++i) lcu[(size_t)i] = h_cu_seqlens[sb.text_begin + i] - base;
    // Row pointers of the SuperBatch's texts (segments are global here).
    e->h_dst.resize((size_t)S);
    const int64_t d = e->desc.d_model;
    for (int64_t s = sb.seg_begin; s < sb.seg_end; ++s) {
      const surge_segment& g = ctx.segs[(size_t)s];
      float* rb = h_part_out[g.partition] + g.row_offset * d;
      for (int64_t j = 0; j < g.count; ++j)
        e->h_dst[(size_t)(g.first_text - sb.text_begin + j)] = (uint64_t)(uintptr_t)(rb + j * d);
    }
    st = encode_chunks(e, S, d_token_ids + base, lcu.data(), stream);
    if (st != SURGE_OK) return st;
  }
  return end_call(e, stream);
}

surge_status surge_encode_all_streamed(surge_encoder* enc, int64_t n_texts,
                                       const int32_t* h_token_ids, const int64_t* h_cu_seqlens,
                                       const int64_t* h_part_offsets, int32_t n_parts,
                                       int64_t b_min, int64_t n_max, int32_t policy, float* h_out,
                                       int32_t overlap, void* compute_stream, void* copy_stream,
                                       double* h_sb_times, int64_t sb_times_cap,
                                       surge_stream_stats* stats) {
  clear_error();
  if (!enc) return fail(SURGE_ERR_INVALID_ARGUMENT, "encoder is NULL");
  if (!h_part_offsets || !h_cu_seqlens) return fail(SURGE_ERR_INVALID_ARGUMENT, "NULL host array");
  if (n_parts < 0) return fail(SURGE_ERR_INVALID_ARGUMENT, "n_parts < 0");
  if (overlap < 0 || overlap > 2) return fail(SURGE_ERR_INVALID_ARGUMENT, "overlap=%d", overlap);
  if (overlap == 1 && compute_stream == copy_stream)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "overlap needs two different streams");
  if (h_sb_times == nullptr && sb_times_cap != 0)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "sb_times_cap > 0 with NULL h_sb_times");
  const int64_t d = enc->desc.d_model;
  // Validate once against per-partition views of h_out (never dereferenced).
  std::vector<float*> views((size_t)n_parts);
  for (int32_t p = 0; p < n_parts; ++p) views[p] = h_out ? h_out + h_part_offsets[p] * d : nullptr;
  int64_t max_tok = 0, max_txt = 0;
  surge_status st = surge_validate_input(&enc->desc, n_texts, h_cu_seqlens, h_part_offsets, n_parts,
                                         b_min, n_max, policy, views.data(), nullptr, &max_txt,
                                         &max_tok);
  if (st != SURGE_OK) return st;
  Plan plan;
  int64_t ns = 0;
  st = make_plan(h_part_offsets, n_parts, b_min, n_max, policy, &plan, &ns);
  if (st != SURGE_OK) return st;
  if (stats) memset(stats, 0, sizeof(*stats));
  if (n_texts == 0) return SURGE_OK;
  if (!h_token_ids) return fail(SURGE_ERR_INVALID_ARGUMENT, "token_ids is NULL");
  if (((uintptr_t)h_out) & 15u) return fail(SURGE_ERR_INVALID_ARGUMENT, "h_out is not 16-byte aligned");
  HIP_TRY(hipSetDevice(enc->device));
  surge_encoder* e = enc;
  hipStream_t cs = (hipStream_t)compute_stream;
  hipStream_t xs = overlap == 1 ? (hipStream_t)copy_stream : cs;
  const bool zero_copy = overlap == 2;
  // Zero copy: the pooling kernel writes the embeddings through the device
  // mapping of h_out, which must be pinned host memory mapped for this
  // device over its whole extent (checked here, before anything runs).
  float* d_out_mapped = nullptr;
  if (zero_copy) {
    const size_t bytes = (size_t)n_texts * (size_t)d * sizeof(float);
    hipPointerAttribute_t a0, a1;
    const bool ok0 = hipPointerGetAttributes(&a0, h_out) == hipSuccess;
    const bool ok1 = ok0 && hipPointerGetAttributes(&a1, (const char*)h_out + bytes - 1) == hipSuccess;
    (void)hipGetLastError();  // a failed query leaves no sticky error behind
    if (!ok1 || a0.type != hipMemoryTypeHost || a1.type != hipMemoryTypeHost ||
        a0.devicePointer == nullptr ||
        (const char*)a1.devicePointer != (const char*)a0.devicePointer + bytes - 1)
      return fail(SURGE_ERR_INVALID_ARGUMENT,
                  "overlap=2 needs h_out in pinned host memory mapped for the device "
                  "(hipHostMalloc) over all %lld rows", (long long)n_texts);
    d_out_mapped = (float*)a0.devicePointer;
  }

  // Staging buffers and events, released on every exit path after both
  // streams have drained.
  struct Res {
    int32_t* tok[2] = {nullptr, nullptr};
    float* out[2] = {nullptr, nullptr};
    std::vector<hipEvent_t> ev;
    hipStream_t s1 = nullptr, s2 = nullptr;
    ~Res() {
      if (s1) hipStreamSynchronize(s1);
      if (s2) hipStreamSynchronize(s2);
      for (int i = 0; i < 2; ++i) {
        if (tok[i]) hipFree(tok[i]);
        if (out[i]) hipFree(out[i]);
      }
      for (hipEvent_t x : ev) hipEventDestroy(x);
    }
  } r;
  r.s1 = cs;
  r.s2 = xs;
  // Lemma 1's staging: per buffer the largest SuperBatch's tokens (int32)
  // and, unless zero copy, its [S, d] fp32 embeddings.
  const int64_t staging =
      2 * (std::max<int64_t>(max_tok, 1) * 4 + (zero_copy ? 0 : max_txt * d * 4));
  for (int i = 0; i < 2; ++i) {
    HIP_TRY(hipMalloc(&r.tok[i], (size_t)std::max<int64_t>(max_tok, 1) * 4));
    if (!zero_copy) HIP_TRY(hipMalloc(&r.out[i], (size_t)max_txt * d * 4));
  }
  // Ordered after the encoder's previous call, on both streams.
  st = begin_call(e, cs);
  if (st != SURGE_OK) return st;
  if (xs != cs) {
    st = begin_call(e, xs);
    if (st != SURGE_OK) return st;
  }
  // Six events per SuperBatch: upload, encode and download start / end.
  r.ev.resize((size_t)ns * 6, nullptr);
  for (hipEvent_t& x : r.ev) HIP_TRY(hipEventCreate(&x));
  auto EV = [&](int64_t j, int k) { return r.ev[(size_t)j * 6 + k]; };
  enum { H2D0, H2D1, ENC0, ENC1, D2H0, D2H1 };

  auto upload = [&](int64_t j) -> surge_status {
    const PlanSB& sb = plan.sbs[(size_t)j];
    const int64_t t0 = h_cu_seqlens[sb.text_begin], t1 = h_cu_seqlens[sb.text_end];
    HIP_TRY(hipEventRecord(EV(j, H2D0), xs));
    HIP_TRY(hipMemcpyAsync(r.tok[j & 1], h_token_ids + t0, (size_t)(t1 - t0) * 4,
                           hipMemcpyHostToDevice, xs));
    HIP_TRY(hipEventRecord(EV(j, H2D1), xs));
    return SURGE_OK;
  };
  auto download = [&](int64_t j) -> surge_status {
    const PlanSB& sb = plan.sbs[(size_t)j];
    const int64_t S = sb.text_end - sb.text_begin;
    HIP_TRY(hipEventRecord(EV(j, D2H0), xs));
    if (!zero_copy)  // (zero copy: the rows are already in h_out)
      HIP_TRY(hipMemcpyAsync(h_out + sb.text_begin * d, r.out[j & 1], (size_t)S * d * 4,
                             hipMemcpyDeviceToHost, xs));
    HIP_TRY(hipEventRecord(EV(j, D2H1), xs));
    return SURGE_OK;
  };
  std::vector<int64_t> lcu;
  st = upload(0);
  if (st != SURGE_OK) return st;
  for (int64_t j = 0; j < ns; ++j) {
    const PlanSB& sb = plan.sbs[(size_t)j];
    const int64_t S = sb.text_end - sb.text_begin;
    if (overlap == 1) {
      HIP_TRY(hipStreamWaitEvent(cs, EV(j, H2D1), 0));
      if (j >= 2) HIP_TRY(hipStreamWaitEvent(cs, EV(j - 2, D2H1), 0));  // staging j&1 is free
    }
    // Rows of this SuperBatch's texts: in the embedding staging buffer, or
    // (zero copy) in the device mapping of h_out.
    e->h_dst.resize((size_t)S);
    for (int64_t i = 0; i < S; ++i)
      e->h_dst[(size_t)i] =
          zero_copy ? (uint64_t)(uintptr_t)(d_out_mapped + (sb.text_begin + i) * d)
                    : (uint64_t)(uintptr_t)(r.out[j & 1] + i * d);
    lcu.resize((size_t)S + 1);
    const int64_t base = h_cu_seqlens[sb.text_begin];
    for (int64_t i = 0; i <= S; ++i) lcu[(size_t)i] = h_cu_seqlens[sb.text_begin + i] - base;
    HIP_TRY(hipEventRecord(EV(j, ENC0), cs));
    st = encode_chunks(e, S, r.tok[j & 1], lcu.data(), cs);
    if (st != SURGE_OK) return st;
    HIP_TRY(hipEventRecord(EV(j, ENC1), cs));
    if (overlap == 1) {
      if (j + 1 < ns) {
        if (j >= 1) HIP_TRY(hipStreamWaitEvent(xs, EV(j - 1, ENC1), 0));  // tokens j+1 & 1 free
        st = upload(j + 1);
        if (st != SURGE_OK) return st;
      }
      HIP_TRY(hipStreamWaitEvent(xs, EV(j, ENC1), 0));
      st = download(j);
      if (st != SURGE_OK) return st;
    } else {
      st = download(j);
      if (st != SURGE_OK) return st;
      if (j + 1 < ns) {
        st = upload(j + 1);
        if (st != SURGE_OK) return st;
      }
    }
  }
  st = end_call(e, xs);  // the copy stream ends last (it waits for the last encode)
  if (st != SURGE_OK) return st;
  HIP_TRY(hipStreamSynchronize(cs));
  HIP_TRY(hipStreamSynchronize(xs));
  // Timing summary.
  auto span = [&](hipEvent_t a, hipEvent_t b) {
    float ms = 0.0f;
    hipEventElapsedTime(&ms, a, b);
    return (double)ms;
  };
  double enc_ms = 0.0, h2d_ms = 0.0, d2h_ms = 0.0;
  for (int64_t j = 0; j < ns; ++j) {
    const double u = span(EV(j, H2D0), EV(j, H2D1));
    const double c = span(EV(j, ENC0), EV(j, ENC1));
    const double w = zero_copy ? 0.0 : span(EV(j, D2H0), EV(j, D2H1));
    h2d_ms += u;
    enc_ms += c;
    d2h_ms += w;
    if (j < sb_times_cap) {
      h_sb_times[3 * j + 0] = u;
      h_sb_times[3 * j + 1] = c;
      h_sb_times[3 * j + 2] = w;
    }
  }
  if (stats) {
    stats->n_superbatches = ns;
    stats->total_ms = span(EV(0, H2D0), EV(ns - 1, D2H1));
    stats->ttfo_ms = span(EV(0, H2D0), EV(0, D2H1));
    stats->enc_ms = enc_ms;
    stats->h2d_ms = h2d_ms;
    stats->d2h_ms = d2h_ms;
    const double io = (h2d_ms + d2h_ms) / (double)ns, ce = enc_ms / (double)ns;
    stats->rho = io > 0.0 ? 1.0 - std::max(0.0, io - ce) / io : 1.0;
    const double exposed = stats->total_ms - enc_ms;
    stats->rho_measured =
        h2d_ms + d2h_ms > 0.0 ? std::min(1.0, std::max(0.0, 1.0 - exposed / (h2d_ms + d2h_ms)))
                              : 1.0;
    stats->staging_bytes = staging;
    stats->max_sb_texts = max_txt;
    stats->max_sb_tokens = max_tok;
  }
  int flag = 0;
  HIP_TRY(hipMemcpy(&flag, e->d_err, sizeof(int), hipMemcpyDeviceToHost));
  if (flag) {
    HIP_TRY(hipMemset(e->d_err, 0, sizeof(int)));
    return fail(SURGE_ERR_INVALID_ARGUMENT, "a token ID outside [0, vocab) was encoded as ID 0");
  }
  return SURGE_OK;
}

surge_status surge_check(surge_encoder* enc, void* hip_stream) {
  clear_error();
  if (!enc) return fail(SURGE_ERR_INVALID_ARGUMENT, "encoder is NULL");
  HIP_TRY(hipSetDevice(enc->device));
  HIP_TRY(hipStreamSynchronize((hipStream_t)hip_stream));
  if (enc->last_use_recorded) HIP_TRY(hipEventSynchronize(enc->last_use));
  int flag = 0;
  HIP_TRY(hipMemcpy(&flag, enc->d_err, sizeof(int), hipMemcpyDeviceToHost));
  if (flag) {
    HIP_TRY(hipMemset(enc->d_err, 0, sizeof(int)));
    return fail(SURGE_ERR_INVALID_ARGUMENT, "a token ID outside [0, vocab) was encoded as ID 0");
  }
  return SURGE_OK;
}

surge_status surge_profile_enable(surge_encoder* enc, int32_t on) {
  return surge_profile_select(enc, on ? (1u << SURGE_KERNEL_COUNT) - 1u : 0u);
}

surge_status surge_profile_select(surge_encoder* enc, uint32_t mask) {
  clear_error();
  if (!enc) return fail(SURGE_ERR_INVALID_ARGUMENT, "encoder is NULL");
  if (mask >> SURGE_KERNEL_COUNT)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "kernel class mask 0x%x has bits above class %d",
                mask, SURGE_KERNEL_COUNT - 1);
  enc->prof_kinds = mask;
  enc->prof_used = 0;
  enc->prof_recs.clear();
  return SURGE_OK;
}

surge_status surge_profile_read(surge_encoder* enc, surge_kernel_stat* stats, int32_t n_stats) {
  clear_error();
  if (!enc || !stats) return fail(SURGE_ERR_INVALID_ARGUMENT, "NULL argument");
  for (int i = 0; i < n_stats; ++i) stats[i] = surge_kernel_stat{0, 0.0, 0.0, 0.0};
  HIP_TRY(hipSetDevice(enc->device));
  for (const ProfRecord& r : enc->prof_recs) {
    if (r.kind >= n_stats) continue;
    HIP_TRY(hipEventSynchronize(enc->prof_events[r.ev + 1]));
    float ms = 0.0f;
    HIP_TRY(hipEventElapsedTime(&ms, enc->prof_events[r.ev], enc->prof_events[r.ev + 1]));
    surge_kernel_stat& s = stats[r.kind];
    s.launches += 1;
    s.total_ms += ms;
    s.flops += r.flops;
    s.bytes += r.bytes;
  }
  return SURGE_OK;
}

}  // extern "C"
