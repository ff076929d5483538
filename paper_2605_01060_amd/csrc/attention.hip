// Packed variable-length self-attention (gfx950, bf16 MFMA, fp32 softmax).
//
// Texts are packed back to back with no padding; text i owns token rows
// cu[i] .. cu[i+1]-1 of the QKV matrix.  Attention is block-diagonal: a
// query attends to the keys of its own text only, bidirectionally, with
// scale 1/sqrt(dh).
//
// One wave handles one (head, text) pair and walks the text in 32-query
// blocks; for each it streams 32-key blocks with an online softmax.  Scores
// are computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16 so that
// every lane owns one query column: the running max, the running sum and the
// rescaling of the output are per-lane scalars, combined with the partner
// lane (lane ^ 32) that holds the other half of the key block.  The
// probabilities stay in registers in exactly the operand layout the P V
// product needs (O^T = V^T P^T), and the V block is staged through LDS so
// each lane can read the 8 keys its MFMA slots stand for.
#include <math.h>

#include "device_common.h"
#include "kernels.h"

namespace surge {
namespace {

template <int DH>
__global__ __launch_bounds__(64) void attention_varlen_kernel(const uint16_t* __restrict__ qkv,
                                                              uint16_t* __restrict__ out,
                                                              const int32_t* __restrict__ cu,
                                                              int n_heads, float scale_log2) {
  constexpr int KSTEPS = DH / 16;       // MFMA steps over the head dimension for S
  constexpr int DT = DH / 32;           // 32-row tiles of O^T
  constexpr int VCHUNKS = 32 * DH / 8;  // 16-byte chunks of a 32-key V block
  __shared__ uint16_t sV[32 * DH];

  const int h = blockIdx.x % n_heads;
  const int t = blockIdx.x / n_heads;
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

  for (int q0 = 0; q0 < L; q0 += 32) {
    const int q = min(q0 + col, L - 1);
    bf16x8 qf[KSTEPS];
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk)
      qf[kk] = as_bf16x8(*reinterpret_cast<const uint4*>(Qb + (size_t)q * ld + kk * 16 + half * 8));

    float m_run = -INFINITY;
    float l_run = 0.0f;
    f32x16 o[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[dt][r] = 0.0f;

    for (int k0 = 0; k0 < L; k0 += 32) {
      // S^T block: rows = keys k0..k0+31 (A operand = K), cols = queries.
      const int kr = min(k0 + col, L - 1);
      f32x16 s;
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = 0.0f;
#pragma unroll
      for (int kk = 0; kk < KSTEPS; ++kk) {
        const bf16x8 kf =
            as_bf16x8(*reinterpret_cast<const uint4*>(Kb + (size_t)kr * ld + kk * 16 + half * 8));
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], s, 0, 0, 0);
      }

      // Stage the V block (rows past the text are read clamped; their
      // probabilities are zero).
#pragma unroll
      for (int c = lane; c < VCHUNKS; c += 64) {
        const int row = c / (DH / 8);
        const int ch = c % (DH / 8);
        const int vr = min(k0 + row, L - 1);
        reinterpret_cast<uint4*>(sV)[c] =
            *(reinterpret_cast<const uint4*>(Vb + (size_t)vr * ld) + ch);
      }

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
      const float alpha = exp2f(m_run - m_new);
      float psum = 0.0f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[r] = exp2f(s[r] - m_new);
        psum += s[r];
      }
      psum += __shfl_xor(psum, 32, 64);
      l_run = l_run * alpha + psum;
      m_run = m_new;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;

      __syncthreads();

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
      __syncthreads();
    }

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
}

}  // namespace

hipError_t launch_attention(const uint16_t* qkv, uint16_t* out, const int32_t* cu, int n_texts,
                            int n_heads, int d_head, hipStream_t stream) {
  if (n_texts <= 0) return hipSuccess;
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)d_head);
  const dim3 grid((unsigned)n_texts * (unsigned)n_heads);
  if (d_head == 64)
    hipLaunchKernelGGL(attention_varlen_kernel<64>, grid, dim3(64), 0, stream, qkv, out, cu,
                       n_heads, scale_log2);
  else
    hipLaunchKernelGGL(attention_varlen_kernel<32>, grid, dim3(64), 0, stream, qkv, out, cu,
                       n_heads, scale_log2);
  return hipGetLastError();
}

}  // namespace surge
