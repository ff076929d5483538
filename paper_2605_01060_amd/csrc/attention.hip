// Packed variable-length self-attention (gfx950, bf16 MFMA, fp32 softmax).
//
// Texts are packed back to back with no padding; text i owns token rows
// cu[i] .. cu[i+1]-1 of the QKV matrix.  Attention is block-diagonal: a
// query attends to the keys of its own text only, bidirectionally, with
// scale 1/sqrt(dh).
//
// Work decomposition.  A work item is (text, 32-query block); the host
// lists the items of a chunk longest text first, so the long texts start
// early and the short ones fill in behind them.  One wave handles one item
// for one head: it walks the text's keys in 32-key blocks with an online
// softmax, prefetching the next block's K fragments and V rows into
// registers while the current block is on the MFMA units.
//
// Scores are computed transposed, S^T = K Q^T, with
// v_mfma_f32_32x32x16_bf16 so that every lane owns one query column: the
// running max, the running sum and the rescaling of the output are per-lane
// scalars, combined with the partner lane (lane ^ 32) that holds the other
// half of the key block.  The probabilities stay in registers in exactly
// the operand layout the P V product needs (O^T = V^T P^T); the V block is
// staged through LDS so each lane can read the keys its MFMA slots stand
// for.
#include <math.h>

#include "device_common.h"
#include "kernels.h"

namespace surge {
namespace {

template <int DH>
__global__ __launch_bounds__(64) void attention_varlen_kernel(const uint16_t* __restrict__ qkv,
                                                              uint16_t* __restrict__ out,
                                                              const int32_t* __restrict__ cu,
                                                              const uint32_t* __restrict__ items,
                                                              int n_heads, float scale_log2) {
  constexpr int KSTEPS = DH / 16;      // MFMA steps over the head dimension for S
  constexpr int DT = DH / 32;          // 32-row tiles of O^T
  constexpr int VCH = 32 * DH / 8;     // 16-byte chunks of a 32-key V block
  constexpr int VPL = VCH / 64;        // ... per lane
  constexpr int CPR = DH / 8;          // 16-byte chunks per V row
  __shared__ uint16_t sV[32 * DH];

  const int h = blockIdx.x % n_heads;
  const uint32_t item = items[blockIdx.x / n_heads];
  const int t = (int)(item >> 7);
  const int q0 = (int)(item & 127u) * 32;
  const int lane = threadIdx.x;
  const int col = lane & 31;
  const int half = lane >> 5;
  const int beg = cu[t];
  const int L = cu[t + 1] - beg;
  const int D = n_heads * DH;
  const size_t ld = (size_t)3 * D;
  const uint16_t* Qb = qkv + (size_t)beg * ld + (size_t)h * DH;
  const uint16_t* Kb = Qb + D;
  const uint16_t* Vb = Qb + 2 * D;

  const int q = min(q0 + col, L - 1);
  bf16x8 qf[KSTEPS];
#pragma unroll
  for (int kk = 0; kk < KSTEPS; ++kk)
    qf[kk] = as_bf16x8(*reinterpret_cast<const uint4*>(Qb + (size_t)q * ld + kk * 16 + half * 8));

  // Prefetch registers for one key block: K fragments (rows = keys) and the
  // lane's share of the V rows (rows past the text are read clamped; their
  // probabilities are zero).
  u32x4 kf[KSTEPS], vr[VPL];
#define SURGE_LOAD_KV_BLOCK(k0_)                                                              \
  do {                                                                                        \
    const int kr_ = min((k0_) + col, L - 1);                                                  \
    _Pragma("unroll") for (int kk = 0; kk < KSTEPS; ++kk) kf[kk] =                            \
        *reinterpret_cast<const u32x4*>(Kb + (size_t)kr_ * ld + kk * 16 + half * 8);          \
    _Pragma("unroll") for (int c = 0; c < VPL; ++c) {                                         \
      const int idx_ = lane + 64 * c;                                                         \
      const int row_ = min((k0_) + idx_ / CPR, L - 1);                                        \
      vr[c] = *(reinterpret_cast<const u32x4*>(Vb + (size_t)row_ * ld) + idx_ % CPR);         \
    }                                                                                         \
  } while (0)
  SURGE_LOAD_KV_BLOCK(0);

  float m_run = -INFINITY;
  float l_run = 0.0f;
  f32x16 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[dt][r] = 0.0f;

  for (int k0 = 0; k0 < L; k0 += 32) {
    // Consume the prefetched block, then start loading the next one.
    bf16x8 kc[KSTEPS];
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) kc[kk] = __builtin_bit_cast(bf16x8, kf[kk]);
    __syncthreads();  // the previous block's P V reads of sV are done
#pragma unroll
    for (int c = 0; c < VPL; ++c) reinterpret_cast<u32x4*>(sV)[lane + 64 * c] = vr[c];
    if (k0 + 32 < L) SURGE_LOAD_KV_BLOCK(k0 + 32);

    // S^T block: rows = keys k0..k0+31 (A operand = K), cols = queries.
    f32x16 s;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = 0.0f;
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk)
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kc[kk], qf[kk], s, 0, 0, 0);

    // Register r holds the score of key k0 + 8*(r/4) + 4*half + r%4.
    float mloc = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = k0 + 8 * (r >> 2) + 4 * half + (r & 3);
      s[r] = key < L ? s[r] * scale_log2 : -INFINITY;
      mloc = fmaxf(mloc, s[r]);
    }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
    const float m_new = fmaxf(m_run, mloc);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    float psum = 0.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      s[r] = __builtin_amdgcn_exp2f(s[r] - m_new);
      psum += s[r];
    }
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;

    __syncthreads();  // sV written

    // O^T += V^T P^T over two 16-key halves c: slot j of this lane is key
    // 16c + 8*(j/4) + 4*half + j%4, the same key for the P (B) and V (A)
    // operands.
    bf16x8 pb[2];
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int j = 0; j < 8; ++j) pb[c][j] = (__bf16)s[8 * c + j];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        bf16x8 va;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int key = 16 * c + 8 * (j >> 2) + 4 * half + (j & 3);
          va[j] = __builtin_bit_cast(__bf16, sV[key * DH + dt * 32 + col]);
        }
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[c], o[dt], 0, 0, 0);
      }
    }
  }

#undef SURGE_LOAD_KV_BLOCK
  // O^T register r of tile dt: head feature dt*32 + 8*(r/4) + 4*half + r%4
  // of query q0 + col.
  if (q0 + col < L) {
    const float inv = 1.0f / l_run;
    uint16_t* orow = out + (size_t)(beg + q0 + col) * D + (size_t)h * DH;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        uint2 w;
        w.x = pack_bf16x2(o[dt][4 * g + 0] * inv, o[dt][4 * g + 1] * inv);
        w.y = pack_bf16x2(o[dt][4 * g + 2] * inv, o[dt][4 * g + 3] * inv);
        *reinterpret_cast<uint2*>(orow + dt * 32 + 8 * g + 4 * half) = w;
      }
    }
  }
}

}  // namespace

hipError_t launch_attention(const uint16_t* qkv, uint16_t* out, const int32_t* cu,
                            const uint32_t* items, int n_items, int n_heads, int d_head,
                            hipStream_t stream) {
  if (n_items <= 0) return hipSuccess;
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)d_head);
  const dim3 grid((unsigned)n_items * (unsigned)n_heads);
  if (d_head == 64)
    hipLaunchKernelGGL(attention_varlen_kernel<64>, grid, dim3(64), 0, stream, qkv, out, cu, items,
                       n_heads, scale_log2);
  else
    hipLaunchKernelGGL(attention_varlen_kernel<32>, grid, dim3(64), 0, stream, qkv, out, cu, items,
                       n_heads, scale_log2);
  return hipGetLastError();
}

int attention_items(const int64_t* cu, int64_t n_texts, uint32_t* items) {
  // (text, query block) pairs, longest text first; ties keep text order.
  int64_t n = 0;
  int64_t maxL = 0;
  for (int64_t i = 0; i < n_texts; ++i) maxL = cu[i + 1] - cu[i] > maxL ? cu[i + 1] - cu[i] : maxL;
  const int64_t max_blocks = (maxL + 31) / 32;
  for (int64_t nb = max_blocks; nb >= 1; --nb) {
    for (int64_t i = 0; i < n_texts; ++i) {
      const int64_t L = cu[i + 1] - cu[i];
      if ((L + 31) / 32 != nb) continue;
      for (int64_t b = 0; b < nb; ++b) items[n++] = (uint32_t)((i << 7) | b);
    }
  }
  return (int)n;
}

}  // namespace surge
