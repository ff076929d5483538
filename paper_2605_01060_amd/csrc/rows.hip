// Row-wise, HBM-bound kernels: embedding gather + LayerNorm, LayerNorm, and
// masked mean pooling + L2 normalisation + partition scatter.
//
// A row of d bf16 values is read as d/8 16-byte chunks spread over the 64
// lanes of one wave (at most two chunks per lane for d <= 1024); mean and
// variance are wave reductions in fp32 (two passes over the registers, so
// the variance is taken about the mean).
#include <math.h>

#include "device_common.h"
#include "kernels.h"

namespace surge {
namespace {

constexpr int MAXC = 2;  // 16-byte chunks per lane, d <= 64 * 2 * 8 = 1024

__device__ __forceinline__ void ln_row(float (&v)[MAXC][8], int nch, int lane, int d,
                                       const float* __restrict__ gamma,
                                       const float* __restrict__ beta, float eps,
                                       uint16_t* __restrict__ yrow) {
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    if (lane + 64 * c < nch) {
#pragma unroll
      for (int e = 0; e < 8; ++e) s += v[c][e];
    }
  }
  const float mean = wave_sum(s) / (float)d;
  float q = 0.0f;
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    if (lane + 64 * c < nch) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float t = v[c][e] - mean;
        q += t * t;
      }
    }
  }
  const float var = wave_sum(q) / (float)d;
  const float rstd = 1.0f / sqrtf(var + eps);
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int ch = lane + 64 * c;
    if (ch < nch) {
      const float4 g0 = reinterpret_cast<const float4*>(gamma)[2 * ch];
      const float4 g1 = reinterpret_cast<const float4*>(gamma)[2 * ch + 1];
      const float4 b0 = reinterpret_cast<const float4*>(beta)[2 * ch];
      const float4 b1 = reinterpret_cast<const float4*>(beta)[2 * ch + 1];
      const float g[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
      const float b[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
      float o[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = (v[c][e] - mean) * rstd * g[e] + b[e];
      reinterpret_cast<uint4*>(yrow)[ch] = pack8(o);
    }
  }
}

// One block per work item (text t, rows 32b .. 32b+31 of it), so a long
// text is spread over several blocks instead of keeping one block busy to
// the end of the launch; the block's four waves take the item's rows in
// turn.  A wave fetches its next row's token ID and table chunks before it
// normalises the current row, so one row's gather latency hides behind the
// previous row's work.
__global__ __launch_bounds__(256) void embed_ln_kernel(
    const int32_t* __restrict__ tokens, const int32_t* __restrict__ cu,
    const uint32_t* __restrict__ items, const uint16_t* __restrict__ word,
    const uint16_t* __restrict__ pos, const float* __restrict__ gamma,
    const float* __restrict__ beta, float eps, int vocab, int d, uint16_t* __restrict__ out,
    int* __restrict__ err) {
  const uint32_t item = items[blockIdx.x];
  const int t = (int)(item >> 7);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int beg = cu[t];
  const int r0 = (int)(item & 127u) * 32;           // first row of the item
  const int r1 = min(r0 + 32, cu[t + 1] - beg);     // one past its last
  const int nch = d >> 3;
  // Table chunks of row p (word row of its checked ID, position row p).
  auto fetch = [&](int p, uint4 (&w)[MAXC], uint4 (&q)[MAXC]) {
    int id = tokens[beg + p];
    if (id < 0 || id >= vocab) {
      if (lane == 0) atomicOr(err, 1);
      id = 0;
    }
    const uint4* wr = reinterpret_cast<const uint4*>(word + (size_t)id * d);
    const uint4* pr = reinterpret_cast<const uint4*>(pos + (size_t)p * d);
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
      const int ch = lane + 64 * c;
      if (ch < nch) {
        w[c] = wr[ch];
        q[c] = pr[ch];
      }
    }
  };
  uint4 wn[MAXC], qn[MAXC];
  if (r0 + wave < r1) fetch(r0 + wave, wn, qn);
  for (int p = r0 + wave; p < r1; p += 4) {
    float v[MAXC][8];
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
      if (lane + 64 * c < nch) {
        float a[8], b[8];
        unpack8(wn[c], a);
        unpack8(qn[c], b);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[c][e] = a[e] + b[e];
      }
    }
    if (p + 4 < r1) fetch(p + 4, wn, qn);
    ln_row(v, nch, lane, d, gamma, beta, eps, out + (size_t)(beg + p) * d);
  }
}

// One wave per row, four rows per block.
__global__ __launch_bounds__(256) void layernorm_kernel(const uint16_t* __restrict__ x,
                                                        const float* __restrict__ gamma,
                                                        const float* __restrict__ beta, float eps,
                                                        uint16_t* __restrict__ y, int64_t M,
                                                        int d) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= M) return;
  const int nch = d >> 3;
  const uint4* xr = reinterpret_cast<const uint4*>(x + (size_t)row * d);
  float v[MAXC][8];
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int ch = lane + 64 * c;
    if (ch < nch) unpack8(xr[ch], v[c]);
  }
  ln_row(v, nch, lane, d, gamma, beta, eps, y + (size_t)row * d);
}

// One block per text: 2 groups of 128 threads split the text's rows, each
// thread owns one 16-byte column chunk; the norm is a block reduction.
// With LN, x holds raw rows and row t's LayerNorm is applied on the fly:
// rows[t] = (rstd, -mean rstd), and the pooled vector is
// gamma * mean_t(x_t rstd_t - mean_t rstd_t) + beta.
template <bool LN>
__global__ __launch_bounds__(256) void pool_l2_scatter_kernel(const uint16_t* __restrict__ x,
                                                              const int32_t* __restrict__ cu,
                                                              const uint64_t* __restrict__ dst,
                                                              int d, const float2* __restrict__ rows,
                                                              const float* __restrict__ gamma,
                                                              const float* __restrict__ beta) {
  __shared__ float part[128 * 8];
  __shared__ float red[4];
  const int t = blockIdx.x;
  const int c = threadIdx.x & 127;
  const int grp = threadIdx.x >> 7;
  const int beg = cu[t];
  const int L = cu[t + 1] - beg;
  const int nch = d >> 3;
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  if (c < nch) {
    // Unrolled so that several rows' loads are in flight at once (the sum
    // keeps its row order).
#pragma unroll 4
    for (int p = grp; p < L; p += 2) {
      float f[8];
      unpack8(reinterpret_cast<const uint4*>(x + (size_t)(beg + p) * d)[c], f);
      if constexpr (LN) {
        const float2 rf = rows[beg + p];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += fmaf(f[e], rf.x, rf.y);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += f[e];
      }
    }
  }
  if (grp == 1 && c < nch) {
#pragma unroll
    for (int e = 0; e < 8; ++e) part[c * 8 + e] = acc[e];
  }
  __syncthreads();
  float sq = 0.0f;
  if (grp == 0 && c < nch) {
    const float invL = 1.0f / (float)L;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      acc[e] = (acc[e] + part[c * 8 + e]) * invL;
      if constexpr (LN) acc[e] = fmaf(acc[e], gamma[8 * c + e], beta[8 * c + e]);
      sq += acc[e] * acc[e];
    }
  }
  sq = wave_sum(sq);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = sq;
  __syncthreads();
  const float norm = sqrtf(red[0] + red[1]);
  const float inv = 1.0f / fmaxf(norm, 1e-12f);
  if (grp == 0 && c < nch) {
    float* row = reinterpret_cast<float*>(dst[t]);
    float4 a = make_float4(acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv);
    float4 b = make_float4(acc[4] * inv, acc[5] * inv, acc[6] * inv, acc[7] * inv);
    reinterpret_cast<float4*>(row)[2 * c] = a;
    reinterpret_cast<float4*>(row)[2 * c + 1] = b;
  }
}

// Per-row LayerNorm factors from equal-width statistics partials (mean,
// biased variance) at stats[p * M + row]: the row's mean is the average of
// the partial means and its variance the average partial variance plus the
// variance of the partial means.  rows[row] = (rstd, -mean * rstd), so that
// LN(v) = gamma (v rstd - mean rstd) + beta.  With MAXP > 0 (parts <= MAXP,
// the encoder's case: d_model / 64 <= 16) every partial is loaded before any
// is used, so the loads' latencies overlap; MAXP = 0 takes any count.  Both
// forms sum in the same order.
template <int MAXP>
__global__ __launch_bounds__(256) void ln_rows_kernel(const float2* __restrict__ stats, int parts,
                                                      int64_t M, float eps,
                                                      float2* __restrict__ rows) {
  const int64_t m = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (m >= M) return;
  float sm = 0.0f, sv = 0.0f, sd = 0.0f;
  const float inv_p = 1.0f / (float)parts;
  if constexpr (MAXP > 0) {
    float2 v[MAXP];
#pragma unroll
    for (int p = 0; p < MAXP; ++p)
      if (p < parts) v[p] = stats[(size_t)p * M + m];
#pragma unroll
    for (int p = 0; p < MAXP; ++p)
      if (p < parts) {
        sm += v[p].x;
        sv += v[p].y;
      }
    const float mu = sm * inv_p;
#pragma unroll
    for (int p = 0; p < MAXP; ++p)
      if (p < parts) {
        const float dm = v[p].x - mu;
        sd = fmaf(dm, dm, sd);
      }
    const float rstd = 1.0f / sqrtf((sv + sd) * inv_p + eps);
    rows[m] = make_float2(rstd, -mu * rstd);
  } else {
    for (int p = 0; p < parts; ++p) {
      const float2 v = stats[(size_t)p * M + m];
      sm += v.x;
      sv += v.y;
    }
    const float mu = sm * inv_p;
    for (int p = 0; p < parts; ++p) {
      const float dm = stats[(size_t)p * M + m].x - mu;
      sd = fmaf(dm, dm, sd);
    }
    const float rstd = 1.0f / sqrtf((sv + sd) * inv_p + eps);
    rows[m] = make_float2(rstd, -mu * rstd);
  }
}

}  // namespace

hipError_t launch_embed_ln(const int32_t* tokens, const int32_t* cu, const uint32_t* items,
                           int n_items, const uint16_t* word, const uint16_t* pos,
                           const float* gamma, const float* beta, float eps, int vocab, int d,
                           uint16_t* out, int* err, hipStream_t stream) {
  if (n_items <= 0) return hipSuccess;
  hipLaunchKernelGGL(embed_ln_kernel, dim3(n_items), dim3(256), 0, stream, tokens, cu, items, word,
                     pos, gamma, beta, eps, vocab, d, out, err);
  return hipGetLastError();
}

hipError_t launch_ln_rows(const float2* stats, int parts, int64_t M, float eps, float2* rows,
                          hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  if (parts < 1) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((M + 255) / 256));
  if (parts <= 16)
    hipLaunchKernelGGL(ln_rows_kernel<16>, grid, dim3(256), 0, stream, stats, parts, M, eps, rows);
  else
    hipLaunchKernelGGL(ln_rows_kernel<0>, grid, dim3(256), 0, stream, stats, parts, M, eps, rows);
  return hipGetLastError();
}

hipError_t launch_layernorm(const uint16_t* x, const float* gamma, const float* beta, float eps,
                            uint16_t* y, int64_t M, int d, hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  const unsigned blocks = (unsigned)((M + 3) / 4);
  hipLaunchKernelGGL(layernorm_kernel, dim3(blocks), dim3(256), 0, stream, x, gamma, beta, eps, y,
                     M, d);
  return hipGetLastError();
}

hipError_t launch_pool_l2_scatter(const uint16_t* x, const int32_t* cu, int n_texts,
                                  const uint64_t* dst, int d, const float2* rows,
                                  const float* gamma, const float* beta, hipStream_t stream) {
  if (n_texts <= 0) return hipSuccess;
  if (rows)
    hipLaunchKernelGGL(pool_l2_scatter_kernel<true>, dim3(n_texts), dim3(256), 0, stream, x, cu,
                       dst, d, rows, gamma, beta);
  else
    hipLaunchKernelGGL(pool_l2_scatter_kernel<false>, dim3(n_texts), dim3(256), 0, stream, x, cu,
                       dst, d, rows, gamma, beta);
  return hipGetLastError();
}

}  // namespace surge
