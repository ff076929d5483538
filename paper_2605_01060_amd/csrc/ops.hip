// Stage-level entry points: one kernel of the encode path on caller buffers.
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "internal.h"
#include "kernels.h"
#include "surge_ops.h"

using namespace surge;

#define HIP_TRY(expr)                                                                     \
  do {                                                                                    \
    hipError_t e_ = (expr);                                                               \
    if (e_ != hipSuccess)                                                                 \
      return fail(e_ == hipErrorOutOfMemory ? SURGE_ERR_OUT_OF_MEMORY : SURGE_ERR_DEVICE, \
                  "%s failed: %s", #expr, hipGetErrorString(e_));                         \
  } while (0)

namespace {

// Device copy of a checked cu_seqlens (int32), freed on scope exit.
struct DeviceCu {
  int32_t* ptr = nullptr;
  ~DeviceCu() {
    if (ptr) hipFree(ptr);
  }
};

surge_status upload_cu(int64_t n_texts, const int64_t* cu, int64_t max_len, DeviceCu* out,
                       int64_t* n_tokens) {
  if (n_texts < 1) return fail(SURGE_ERR_INVALID_ARGUMENT, "n_texts=%lld < 1", (long long)n_texts);
  if (!cu) return fail(SURGE_ERR_INVALID_ARGUMENT, "cu_seqlens is NULL");
  if (cu[0] != 0) return fail(SURGE_ERR_INVALID_ARGUMENT, "cu_seqlens[0] != 0");
  for (int64_t i = 0; i < n_texts; ++i) {
    const int64_t L = cu[i + 1] - cu[i];
    if (L < 1 || L > max_len)
      return fail(SURGE_ERR_INVALID_ARGUMENT, "text %lld length %lld outside [1, %lld]",
                  (long long)i, (long long)L, (long long)max_len);
  }
  if (cu[n_texts] > (int64_t)INT32_MAX) return fail(SURGE_ERR_INVALID_ARGUMENT, "too many tokens");
  std::vector<int32_t> h((size_t)n_texts + 1);
  for (int64_t i = 0; i <= n_texts; ++i) h[(size_t)i] = (int32_t)cu[i];
  HIP_TRY(hipMalloc(&out->ptr, h.size() * 4));
  HIP_TRY(hipMemcpy(out->ptr, h.data(), h.size() * 4, hipMemcpyHostToDevice));
  *n_tokens = cu[n_texts];
  return SURGE_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Scratch of surge_op_linear_ln_noalloc: the per-row LayerNorm factors of at
// most kScratchRows rows (4 MiB), held by every GPU the library runs on until
// the process ends.  In host code `scratch` names a host-side stand-in, not
// device memory: host code uses only the per-device address obtained from
// hipGetSymbolAddress below.
constexpr int64_t kScratchRows = 1 << 19;
static __device__ __align__(256) float2 scratch[kScratchRows];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float2* g_scratch_ptr[kMaxDevices] = {};

// The device address of the current device's scratch, looked up once per
// device with that device current.
surge_status scratch_address(float2** out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(SURGE_ERR_DEVICE, "device index %d outside [0, %d)", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(SURGE_ERR_DEVICE, "hipGetSymbolAddress returned NULL");
    g_scratch_ptr[dev] = (float2*)p;
  }
  *out = g_scratch_ptr[dev];
  return SURGE_OK;
}

}  // namespace

extern "C" {

surge_status surge_op_embed_ln(int64_t n_texts, const int64_t* cu, const int32_t* d_tokens,
                               const uint16_t* d_word, int32_t vocab, const uint16_t* d_pos,
                               int32_t max_pos, const float* d_gamma, const float* d_beta,
                               float eps, int32_t d, uint16_t* d_out, void* hip_stream) {
  clear_error();
  if (d < 128 || d > 1024 || d % 128) return fail(SURGE_ERR_INVALID_ARGUMENT, "d=%d", d);
  if (vocab < 1 || max_pos < 1) return fail(SURGE_ERR_INVALID_ARGUMENT, "vocab/max_pos < 1");
  if (!d_tokens || !d_word || !d_pos || !d_gamma || !d_beta || !d_out)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "NULL device pointer");
  if (!aligned16(d_word) || !aligned16(d_pos) || !aligned16(d_gamma) || !aligned16(d_beta) ||
      !aligned16(d_out))
    return fail(SURGE_ERR_INVALID_ARGUMENT, "device buffers must be 16-byte aligned");
  DeviceCu dcu;
  int64_t T = 0;
  surge_status st = upload_cu(n_texts, cu, std::min(max_pos, 4096), &dcu, &T);
  if (st != SURGE_OK) return st;
  std::vector<uint32_t> items((size_t)T);
  const int n_items = row_block_items(cu, n_texts, items.data());
  DeviceCu ditems;
  HIP_TRY(hipMalloc(&ditems.ptr, (size_t)n_items * 4));
  HIP_TRY(hipMemcpy(ditems.ptr, items.data(), (size_t)n_items * 4, hipMemcpyHostToDevice));
  int* derr = nullptr;
  HIP_TRY(hipMalloc(&derr, sizeof(int)));
  DeviceCu guard;  // frees derr through the same path
  guard.ptr = (int32_t*)derr;
  HIP_TRY(hipMemset(derr, 0, sizeof(int)));
  hipStream_t s = (hipStream_t)hip_stream;
  HIP_TRY(launch_embed_ln(d_tokens, dcu.ptr, (const uint32_t*)ditems.ptr, n_items, d_word, d_pos,
                          d_gamma, d_beta, eps, vocab, d, d_out, derr, s));
  HIP_TRY(hipStreamSynchronize(s));
  int flag = 0;
  HIP_TRY(hipMemcpy(&flag, derr, sizeof(int), hipMemcpyDeviceToHost));
  if (flag) return fail(SURGE_ERR_INVALID_ARGUMENT, "a token ID outside [0, vocab) was read as 0");
  return SURGE_OK;
}

surge_status surge_op_linear(int64_t M, int32_t N, int32_t K, const uint16_t* d_x,
                             const uint16_t* d_w, const float* d_bias, const uint16_t* d_res,
                             int32_t epilogue, uint16_t* d_y, void* hip_stream) {
  clear_error();
  if (M < 1 || M > (int64_t)INT32_MAX) return fail(SURGE_ERR_INVALID_ARGUMENT, "M=%lld", (long long)M);
  if (N < 128 || N % 128) return fail(SURGE_ERR_INVALID_ARGUMENT, "N=%d not a multiple of 128", N);
  if (K < 64 || K % 64) return fail(SURGE_ERR_INVALID_ARGUMENT, "K=%d not a multiple of 64", K);
  if (epilogue < 0 || epilogue > 2) return fail(SURGE_ERR_INVALID_ARGUMENT, "epilogue=%d", epilogue);
  if (!d_x || !d_w || !d_bias || !d_y || (epilogue == 2 && !d_res))
    return fail(SURGE_ERR_INVALID_ARGUMENT, "NULL device pointer");
  if (!aligned16(d_x) || !aligned16(d_w) || !aligned16(d_bias) || !aligned16(d_y) ||
      (d_res && !aligned16(d_res)))
    return fail(SURGE_ERR_INVALID_ARGUMENT, "device buffers must be 16-byte aligned");
  hipStream_t s = (hipStream_t)hip_stream;
  HIP_TRY(launch_linear(d_x, d_w, d_bias, d_res, d_y, M, N, K, epilogue, LinearExtra(), s));
  HIP_TRY(hipStreamSynchronize(s));
  return SURGE_OK;
}

}  // extern "C"

namespace {

// Argument check shared by surge_op_linear_ln and its no-allocation variant;
// *rows is set when the epilogue reads per-row LayerNorm factors.
surge_status check_linear_ln(int64_t M, int32_t N, int32_t K, const uint16_t* d_x,
                             const uint16_t* d_w, const float* d_bias, const uint16_t* d_res,
                             int32_t epilogue, const float* d_stats_in, int32_t parts_in,
                             const float* d_col_s, const float* d_gamma, const float* d_beta,
                             float eps, float* d_stats_out, uint16_t* d_y, bool* rows) {
  if (M < 1 || M > (int64_t)INT32_MAX) return fail(SURGE_ERR_INVALID_ARGUMENT, "M=%lld", (long long)M);
  if (N < 128 || N % 128) return fail(SURGE_ERR_INVALID_ARGUMENT, "N=%d not a multiple of 128", N);
  if (K < 64 || K % 64) return fail(SURGE_ERR_INVALID_ARGUMENT, "K=%d not a multiple of 64", K);
  if (epilogue < 0 || epilogue > 6) return fail(SURGE_ERR_INVALID_ARGUMENT, "epilogue=%d", epilogue);
  const bool fold = epilogue == EPI_FOLD || epilogue == EPI_FOLD_GELU;
  const bool res = epilogue == EPI_BIAS_RESIDUAL || epilogue >= EPI_RES_STATS;
  const bool lnres = epilogue == EPI_LNRES_STATS;
  const bool stats = epilogue >= EPI_RES_STATS;
  if (!d_x || !d_w || !d_bias || !d_y || (res && !d_res))
    return fail(SURGE_ERR_INVALID_ARGUMENT, "NULL device pointer");
  if ((fold || lnres) && (!d_stats_in || parts_in < 1 || parts_in > 1024))
    return fail(SURGE_ERR_INVALID_ARGUMENT, "stats_in NULL or parts_in=%d outside [1, 1024]",
                parts_in);
  if (fold && !d_col_s) return fail(SURGE_ERR_INVALID_ARGUMENT, "col_s is NULL");
  if (lnres && (!d_gamma || !d_beta)) return fail(SURGE_ERR_INVALID_ARGUMENT, "gamma/beta NULL");
  if (stats && !d_stats_out) return fail(SURGE_ERR_INVALID_ARGUMENT, "stats_out is NULL");
  if ((fold || lnres) && !(eps > 0.0f)) return fail(SURGE_ERR_INVALID_ARGUMENT, "eps must be > 0");
  if (!aligned16(d_x) || !aligned16(d_w) || !aligned16(d_bias) || !aligned16(d_y) ||
      (d_res && !aligned16(d_res)) || (d_col_s && !aligned16(d_col_s)) ||
      (d_gamma && !aligned16(d_gamma)) || (d_beta && !aligned16(d_beta)) ||
      (d_stats_in && ((uintptr_t)d_stats_in & 7u)) || (d_stats_out && ((uintptr_t)d_stats_out & 7u)))
    return fail(SURGE_ERR_INVALID_ARGUMENT, "device buffers must be aligned (16 B; stats 8 B)");
  *rows = fold || lnres;
  return SURGE_OK;
}

// Enqueue the row factors (when `rows` is not NULL) and the linear layer.
surge_status enqueue_linear_ln(int64_t M, int32_t N, int32_t K, const uint16_t* d_x,
                               const uint16_t* d_w, const float* d_bias, const uint16_t* d_res,
                               int32_t epilogue, const float* d_stats_in, int32_t parts_in,
                               const float* d_col_s, const float* d_gamma, const float* d_beta,
                               float eps, float* d_stats_out, uint16_t* d_y, float2* rows,
                               hipStream_t s) {
  LinearExtra ex;
  ex.stats_out = (float2*)d_stats_out;
  ex.col_s = d_col_s;
  ex.gamma = d_gamma;
  ex.beta = d_beta;
  if (rows) {
    HIP_TRY(launch_ln_rows((const float2*)d_stats_in, parts_in, M, eps, rows, s));
    ex.rows_in = rows;
  }
  HIP_TRY(launch_linear(d_x, d_w, d_bias, d_res, d_y, M, N, K, epilogue, ex, s));
  return SURGE_OK;
}

}  // namespace

extern "C" {

surge_status surge_op_linear_ln(int64_t M, int32_t N, int32_t K, const uint16_t* d_x,
                                const uint16_t* d_w, const float* d_bias, const uint16_t* d_res,
                                int32_t epilogue, const float* d_stats_in, int32_t parts_in,
                                const float* d_col_s, const float* d_gamma, const float* d_beta,
                                float eps, float* d_stats_out, uint16_t* d_y, void* hip_stream) {
  clear_error();
  bool need_rows = false;
  surge_status st = check_linear_ln(M, N, K, d_x, d_w, d_bias, d_res, epilogue, d_stats_in,
                                    parts_in, d_col_s, d_gamma, d_beta, eps, d_stats_out, d_y,
                                    &need_rows);
  if (st != SURGE_OK) return st;
  hipStream_t s = (hipStream_t)hip_stream;
  DeviceCu rows;  // per-row LayerNorm factors, freed on return
  if (need_rows) HIP_TRY(hipMalloc(&rows.ptr, (size_t)M * 8));
  st = enqueue_linear_ln(M, N, K, d_x, d_w, d_bias, d_res, epilogue, d_stats_in, parts_in, d_col_s,
                         d_gamma, d_beta, eps, d_stats_out, d_y, (float2*)rows.ptr, s);
  if (st != SURGE_OK) return st;
  HIP_TRY(hipStreamSynchronize(s));
  return SURGE_OK;
}

surge_status surge_op_linear_ln_noalloc(int64_t M, int32_t N, int32_t K, const uint16_t* d_x,
                                        const uint16_t* d_w, const float* d_bias,
                                        const uint16_t* d_res, int32_t epilogue,
                                        const float* d_stats_in, int32_t parts_in,
                                        const float* d_col_s, const float* d_gamma,
                                        const float* d_beta, float eps, float* d_stats_out,
                                        uint16_t* d_y, void* hip_stream) {
  clear_error();
  bool need_rows = false;
  surge_status st = check_linear_ln(M, N, K, d_x, d_w, d_bias, d_res, epilogue, d_stats_in,
                                    parts_in, d_col_s, d_gamma, d_beta, eps, d_stats_out, d_y,
                                    &need_rows);
  if (st != SURGE_OK) return st;
  float2* rows = nullptr;
  if (need_rows) {
    if (M > kScratchRows)
      return fail(SURGE_ERR_CAPACITY, "M=%lld rows exceed the %lld rows of the static scratch",
                  (long long)M, (long long)kScratchRows);
    st = scratch_address(&rows);
    if (st != SURGE_OK) return st;
  }
  return enqueue_linear_ln(M, N, K, d_x, d_w, d_bias, d_res, epilogue, d_stats_in, parts_in,
                           d_col_s, d_gamma, d_beta, eps, d_stats_out, d_y, rows,
                           (hipStream_t)hip_stream);
}

int32_t surge_op_linear_stats_width(int64_t M, int32_t N) { return linear_stats_width(M, N); }

surge_status surge_op_attention(int64_t n_texts, const int64_t* cu, int32_t n_heads, int32_t d_head,
                                const uint16_t* d_qkv, uint16_t* d_out, void* hip_stream) {
  clear_error();
  if (d_head != 32 && d_head != 64) return fail(SURGE_ERR_INVALID_ARGUMENT, "d_head=%d", d_head);
  if (n_heads < 1 || (n_heads * d_head) % 128)
    return fail(SURGE_ERR_INVALID_ARGUMENT, "n_heads*d_head must be a multiple of 128");
  if (!d_qkv || !d_out) return fail(SURGE_ERR_INVALID_ARGUMENT, "NULL device pointer");
  if (!aligned16(d_qkv) || !aligned16(d_out))
    return fail(SURGE_ERR_INVALID_ARGUMENT, "device buffers must be 16-byte aligned");
  DeviceCu dcu;
  int64_t T = 0;
  surge_status st = upload_cu(n_texts, cu, 4096, &dcu, &T);
  if (st != SURGE_OK) return st;
  std::vector<uint32_t> items((size_t)T);
  const int n_items = row_block_items(cu, n_texts, items.data());
  DeviceCu ditems;
  HIP_TRY(hipMalloc(&ditems.ptr, (size_t)n_items * 4));
  HIP_TRY(hipMemcpy(ditems.ptr, items.data(), (size_t)n_items * 4, hipMemcpyHostToDevice));
  hipStream_t s = (hipStream_t)hip_stream;
  HIP_TRY(launch_attention(d_qkv, d_out, dcu.ptr, (const uint32_t*)ditems.ptr, n_items, n_heads,
                           d_head, s));
  HIP_TRY(hipStreamSynchronize(s));
  return SURGE_OK;
}

surge_status surge_op_layernorm(int64_t M, int32_t d, const uint16_t* d_x, const float* d_gamma,
                                const float* d_beta, float eps, uint16_t* d_y, void* hip_stream) {
  clear_error();
  if (M < 1) return fail(SURGE_ERR_INVALID_ARGUMENT, "M < 1");
  if (d < 8 || d > 1024 || d % 8) return fail(SURGE_ERR_INVALID_ARGUMENT, "d=%d", d);
  if (!d_x || !d_gamma || !d_beta || !d_y) return fail(SURGE_ERR_INVALID_ARGUMENT, "NULL pointer");
  if (!aligned16(d_x) || !aligned16(d_gamma) || !aligned16(d_beta) || !aligned16(d_y))
    return fail(SURGE_ERR_INVALID_ARGUMENT, "device buffers must be 16-byte aligned");
  hipStream_t s = (hipStream_t)hip_stream;
  HIP_TRY(launch_layernorm(d_x, d_gamma, d_beta, eps, d_y, M, d, s));
  HIP_TRY(hipStreamSynchronize(s));
  return SURGE_OK;
}

surge_status surge_op_pool_l2(int64_t n_texts, const int64_t* cu, int32_t d, const uint16_t* d_x,
                              float* d_out, void* hip_stream) {
  clear_error();
  if (d < 128 || d > 1024 || d % 128) return fail(SURGE_ERR_INVALID_ARGUMENT, "d=%d", d);
  if (!d_x || !d_out) return fail(SURGE_ERR_INVALID_ARGUMENT, "NULL device pointer");
  if (!aligned16(d_x) || !aligned16(d_out))
    return fail(SURGE_ERR_INVALID_ARGUMENT, "device buffers must be 16-byte aligned");
  DeviceCu dcu;
  int64_t T = 0;
  surge_status st = upload_cu(n_texts, cu, 1 << 16, &dcu, &T);
  if (st != SURGE_OK) return st;
  std::vector<uint64_t> rows((size_t)n_texts);
  for (int64_t i = 0; i < n_texts; ++i) rows[(size_t)i] = (uint64_t)(uintptr_t)(d_out + i * d);
  DeviceCu drows;
  HIP_TRY(hipMalloc(&drows.ptr, rows.size() * 8));
  HIP_TRY(hipMemcpy(drows.ptr, rows.data(), rows.size() * 8, hipMemcpyHostToDevice));
  hipStream_t s = (hipStream_t)hip_stream;
  HIP_TRY(launch_pool_l2_scatter(d_x, dcu.ptr, (int)n_texts, (const uint64_t*)drows.ptr, d,
                                 nullptr, nullptr, nullptr, s));
  HIP_TRY(hipStreamSynchronize(s));
  return SURGE_OK;
}

}  // extern "C"
