// Packed variable-length self-attention (gfx950, bf16 MFMA, fp32 softmax).
//
// Texts are packed back to back with no padding; text i owns token rows
// cu[i] .. cu[i+1]-1 of the QKV matrix.  Attention is block-diagonal: a
// query attends to the keys of its own text only, bidirectionally, with
// scale 1/sqrt(dh).
//
// Work decomposition.  A work item is (text, 32-query block); the host
// lists the items of a chunk longest text first, so the long texts start
// early and the short ones fill in behind them.  One wave (a workgroup of
// its own) handles one item for one head: it walks the text's keys in
// 32-key blocks with an online softmax.
//
// Memory path.  A head's slice of a token row is DH contiguous bf16 (128 B
// for DH = 64).  Q, K and V blocks move from global memory to LDS with
// direct copies that read whole rows (8 lanes per 128-byte row), stored in
// the conflict-free chunk swizzle; the next K/V block is copied into the
// second LDS buffer while the current one is on the MFMA units.  The output
// block is staged in LDS and written back as whole rows too.  (Reading the
// MFMA operands straight from global memory would touch 32 rows per
// instruction for 32 bytes each, which stalls the address path.)
//
// Scores are computed transposed, S^T = K Q^T, with
// v_mfma_f32_32x32x16_bf16 so that every lane owns one query column: the
// running max, the running sum and the rescaling of the output are per-lane
// scalars, combined with the partner lane (lane ^ 32) that holds the other
// half of the key block.  The probabilities stay in registers in exactly
// the operand layout the P V product needs (O^T = V^T P^T); its V^T operand
// is read from the row-major V block with the gfx950 transposing LDS read
// (ds_read_b64_tr_b16), which hands each lane one feature of 4 consecutive
// keys.
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
  constexpr int KSTEPS = DH / 16;  // MFMA steps over the head dimension for S
  constexpr int DT = DH / 32;      // 32-row tiles of O^T
  constexpr int CPR = DH / 8;      // 16-byte chunks per row
  constexpr int RPC = 64 / CPR;    // rows one wave copy fills
  constexpr int NCP = 32 / RPC;    // copies per 32-row block
  constexpr int BLK = 32 * CPR;    // 16-byte slots per 32-row block
  // Two K/V buffers.  The Q block passes through the second K buffer before
  // the first prefetch, and the output block is staged in the first one.
  __shared__ u32x4 sK[2][BLK];
  __shared__ u32x4 sV[2][BLK];
  u32x4* const sQ = sK[1];
  u32x4* const sO = sK[0];

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
  const int ld = 3 * D;
  const uint16_t* Qb = qkv + (size_t)beg * ld + (size_t)h * DH;
  const uint16_t* Kb = Qb + D;
  const uint16_t* Vb = Qb + 2 * D;

  // Copy j of a 32-row block starting at row r0: lane l fills slot
  // j*64 + l, i.e. row r0 + j*RPC + l/CPR with its swizzled chunk.  Rows past
  // the text are read clamped (their scores are masked, their outputs not
  // stored).
  const int crow = lane / CPR;
#define SURGE_COPY_BLOCK(src_, r0_, lds_)                                                   \
  do {                                                                                      \
    _Pragma("unroll") for (int j = 0; j < NCP; ++j) {                                       \
      const int row_ = min((r0_) + j * RPC + crow, L - 1);                                  \
      copy_to_lds16((src_) + __umul24(row_, ld) + copy_chunk<CPR>(lane, j) * 8,             \
                    (lds_) + j * 1024);                                                     \
    }                                                                                       \
  } while (0)

  const uint32_t lq = lds_address(sK[1]);
  const uint32_t lk = lds_address(sK[0]);
  const uint32_t lv = lds_address(sV[0]);
  constexpr uint32_t BUF = BLK * 16;
  SURGE_COPY_BLOCK(Qb, q0, lq);
  SURGE_COPY_BLOCK(Kb, 0, lk);
  SURGE_COPY_BLOCK(Vb, 0, lv);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  bf16x8 qf[KSTEPS];
#pragma unroll
  for (int kk = 0; kk < KSTEPS; ++kk)
    qf[kk] = __builtin_bit_cast(bf16x8, sQ[swz<CPR>(col, kk * 2 + half)]);
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // Q is in registers: sK[1] is free

  // Transposing V reads: lane l supplies the address of 4 features of key
  // 4*half + (l%16)/4 (+ 8 for the second read, + 16c) starting at feature
  // dt*32 + 16*((l/16)%2) + 4*(l%4), and receives feature dt*32 + l%32 of
  // the 4 keys 4*half + 4i..4i+3 of its 16-lane group, i.e. operand slots
  // 4i..4i+3 of key 16c + 8i + 4*half + 0..3.
  const int tr_key = 4 * half + ((lane & 15) >> 2);
  const int tr_feat = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  float m_run = -INFINITY;  // running max, log2 units (raw score x scale_log2)
  float l_run = 0.0f;
  f32x16 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[dt][r] = 0.0f;

  int b = 0;
  for (int k0 = 0; k0 < L; k0 += 32) {
    if (k0 > 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // block k0 is in LDS
    if (k0 + 32 < L) {
      // The other buffer's reads (previous block) were consumed by MFMAs.
      SURGE_COPY_BLOCK(Kb, k0 + 32, lk + (b ^ 1) * BUF);
      SURGE_COPY_BLOCK(Vb, k0 + 32, lv + (b ^ 1) * BUF);
    }
    const u32x4* kb = sK[b];
    const u32x4* vb = sV[b];

    // S^T block: rows = keys k0..k0+31 (A operand = K), cols = queries.
    f32x16 s;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = 0.0f;
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk)
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
          __builtin_bit_cast(bf16x8, kb[swz<CPR>(col, kk * 2 + half)]), qf[kk], s, 0, 0, 0);

    // Register r holds the score of key k0 + 8*(r/4) + 4*half + r%4; only
    // the text's last block has keys past its end (uniform branch).
    if (k0 + 32 > L) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (k0 + 8 * (r >> 2) + 4 * half + (r & 3) >= L) s[r] = -INFINITY;
    }
    float mloc = s[0];
#pragma unroll
    for (int r = 1; r < 16; ++r) mloc = fmaxf(mloc, s[r]);
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
    const float m_new = fmaxf(m_run, mloc * scale_log2);
    float psum = 0.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      s[r] = __builtin_amdgcn_exp2f(fmaf(s[r], scale_log2, -m_new));
      psum += s[r];
    }
    psum += __shfl_xor(psum, 32, 64);
    if (k0 == 0) {
      l_run = psum;  // o is still zero: nothing to rescale
    } else {
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      l_run = fmaf(l_run, alpha, psum);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
    }
    m_run = m_new;

    // O^T += V^T P^T over two 16-key halves c: slot j of this lane is key
    // 16c + 8*(j/4) + 4*half + j%4, the same key for the P (B) and V (A)
    // operands.
    bf16x8 pb[2];
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int j = 0; j < 8; ++j) pb[c][j] = (__bf16)s[8 * c + j];
    const char* vbytes = reinterpret_cast<const char*>(vb);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const int feat = dt * 32 + tr_feat;
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        bf16x4 v2[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          const int key = 16 * c + 8 * i + tr_key;
          const char* pa = vbytes + swz<CPR>(key, feat >> 3) * 16 + (feat & 7) * 2;
          v2[i] = __builtin_bit_cast(bf16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                                 (__attribute__((address_space(3))) i16x4*)pa));
        }
        const bf16x8 va = __builtin_shufflevector(v2[0], v2[1], 0, 1, 2, 3, 4, 5, 6, 7);
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[c], o[dt], 0, 0, 0);
      }
    }
    b ^= 1;
  }
#undef SURGE_COPY_BLOCK

  // O^T register r of tile dt: head feature dt*32 + 8*(r/4) + 4*half + r%4
  // of query q0 + col.  Stage the normalised bf16 block in LDS (row =
  // query), then store whole rows.  All reads of the K/V buffers are done:
  // their results went into MFMAs.
  const float inv = 1.0f / l_run;
  char* obytes = reinterpret_cast<char*>(sO);
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      uint2 w;
      w.x = pack_bf16x2(o[dt][4 * g + 0] * inv, o[dt][4 * g + 1] * inv);
      w.y = pack_bf16x2(o[dt][4 * g + 2] * inv, o[dt][4 * g + 3] * inv);
      *reinterpret_cast<uint2*>(obytes + swz<CPR>(col, dt * 4 + g) * 16 + half * 8) = w;
    }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  uint16_t* ob = out + (size_t)(beg + q0) * D + (size_t)h * DH;
#pragma unroll
  for (int j = 0; j < NCP; ++j) {
    const int row = j * RPC + crow;
    const u32x4 v = sO[j * 64 + lane];
    if (q0 + row < L)
      *reinterpret_cast<u32x4*>(ob + (size_t)row * D + copy_chunk<CPR>(lane, j) * 8) = v;
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
