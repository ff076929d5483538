// Packed variable-length self-attention (gfx950, bf16 MFMA, fp32 softmax).
//
// Texts are packed back to back with no padding; text i owns token rows
// cu[i] .. cu[i+1]-1 of the QKV matrix.  Attention is block-diagonal: a
// query attends to the keys of its own text only, bidirectionally, with
// scale 1/sqrt(dh).
//
// Work decomposition.  A work item is (text, 32-query block); the host
// lists the items of a chunk longest text first, so the long texts start
// early and the short ones fill in behind them.  A unit is one item for one
// head (or head pair, below); a wave (a workgroup of its own) handles UNITS_PER_WAVE units,
// grid-strided, walking each unit's keys in 32-key blocks with an online
// softmax.
//
// Pipelining.  The wave's key blocks form one sequence across its units:
// while block j is on the MFMA units, block j+1 is copied into the other
// buffer, and at a unit's last block that is the next unit's first K/V block
// together with its Q block.  A unit's output block is staged in the K
// buffer of its last key block and stored once the next unit's first block
// has arrived, so every wait is for "everything issued so far" and no wait
// depends on how many stores were issued.
//
// Memory path.  A unit's slice of a token row is 64 contiguous bf16, 128
// bytes (one 64-dimensional head, or a pair of 32-dimensional heads as
// below).  Q, K and V blocks move from global memory to LDS with
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
//
// Head pairs.  With 32-dimensional heads a head's slice of a row is only
// 64 bytes, half a cache line, and a block step has half the MFMA work of a
// 64-dimensional head for the same softmax work.  So a unit then takes two
// adjacent heads: its rows are the pair's 128 contiguous bytes, laid out and
// copied exactly like one 64-dimensional head, while scores, softmax
// statistics and outputs stay separate per head (each head's arithmetic is
// the one-head arithmetic, in the same order), and the wave has two
// independent softmax chains to interleave.
#include <math.h>

#include "device_common.h"
#include "kernels.h"

namespace surge {
namespace {

// Units per wave: enough that most units start on a block copied during
// the previous unit, few enough that the dispatcher still balances the
// uneven unit costs across CUs (measured best at 4 on the bge workload).
constexpr int UNITS_PER_WAVE = 4;

// DH: bytes / 2 of a unit's row slice (64: one 64-dimensional head or, with
// PAIR, two adjacent 32-dimensional heads); n_heads counts such slices.
template <int DH, bool PAIR>
__global__ __launch_bounds__(64) void attention_varlen_kernel(const uint16_t* __restrict__ qkv,
                                                              uint16_t* __restrict__ out,
                                                              const int32_t* __restrict__ cu,
                                                              const uint32_t* __restrict__ items,
                                                              int n_heads, float scale_log2,
                                                              int n_units) {
  constexpr int KSTEPS = DH / 16;  // MFMA steps over the row slice
  constexpr int DT = DH / 32;      // 32-row tiles of O^T
  constexpr int NH = PAIR ? 2 : 1; // heads per unit
  constexpr int KS = KSTEPS / NH;  // MFMA steps over one head for S
  static_assert(!PAIR || DT == NH, "a head pair owns one O^T tile per head");
  constexpr int CPR = DH / 8;      // 16-byte chunks per row
  constexpr int RPC = 64 / CPR;    // rows one wave copy fills
  constexpr int NCP = 32 / RPC;    // copies per 32-row block
  constexpr int BLK = 32 * CPR;    // 16-byte slots per 32-row block
  // Two K/V buffers (block j of the wave's block sequence in buffer j % 2)
  // and the Q block of the next unit.  A unit's output block is staged in
  // the K buffer of its last key block.
  __shared__ u32x4 sK[2][BLK];
  __shared__ u32x4 sV[2][BLK];
  __shared__ u32x4 sQ[BLK];

  const int lane = threadIdx.x;
  const int col = lane & 31;
  const int half = lane >> 5;
  const int D = n_heads * DH;
  const int ld = 3 * D;
  const int crow = lane / CPR;
  const uint32_t lq = lds_address(sQ);
  const uint32_t lk = lds_address(sK[0]);
  const uint32_t lv = lds_address(sV[0]);
  constexpr uint32_t BUF = BLK * 16;

  // A unit is (work item, row slice h): item = (text << 7 | 32-query block).
  struct Unit {
    const uint16_t* base;  // Q row of the text's first token, slice h
    int q0, L, beg, h;
  };
  auto unit_at = [&](int u) {
    Unit r;
    r.h = u % n_heads;
    const uint32_t item = items[u / n_heads];
    const int t = (int)(item >> 7);
    r.q0 = (int)(item & 127u) * 32;
    r.beg = cu[t];
    r.L = cu[t + 1] - r.beg;
    r.base = qkv + (size_t)r.beg * ld + (size_t)r.h * DH;
    return r;
  };
  // Copy j of a 32-row block starting at row r0: lane l fills slot
  // j*64 + l, i.e. row r0 + j*RPC + l/CPR with its swizzled chunk.  Rows past
  // the text are read clamped (their scores are masked, their outputs not
  // stored).
  auto copy_block = [&](const uint16_t* src, int r0, int L, uint32_t lds) {
#pragma unroll
    for (int j = 0; j < NCP; ++j) {
      const int row = min(r0 + j * RPC + crow, L - 1);
      copy_to_lds16(src + __umul24(row, ld) + copy_chunk<CPR>(lane, j) * 8, lds + j * 1024);
    }
  };

  // Transposing V reads: lane l supplies the address of 4 features of key
  // 4*half + (l%16)/4 (+ 8 for the second read, + 16c) starting at feature
  // dt*32 + 16*((l/16)%2) + 4*(l%4), and receives feature dt*32 + l%32 of
  // the 4 keys 4*half + 4i..4i+3 of its 16-lane group, i.e. operand slots
  // 4i..4i+3 of key 16c + 8i + 4*half + 0..3.
  const int tr_key = 4 * half + ((lane & 15) >> 2);
  const int tr_feat = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  const int G = gridDim.x;
  int u = blockIdx.x;  // < n_units: the grid is never larger
  Unit cur = unit_at(u);
  copy_block(cur.base, cur.q0, cur.L, lq);
  copy_block(cur.base + D, 0, cur.L, lk);
  copy_block(cur.base + 2 * D, 0, cur.L, lv);

  int b = 0;                      // buffer of the key block being computed
  bool pending = false;           // a staged output block waits to be stored
  uint16_t* p_ob = nullptr;       // its destination (first query row, head)
  int p_rows = 0;                 // and its valid query rows

  for (;;) {
    const int nkb = (cur.L + 31) / 32;
    const int un = u + G;
    const bool has_next = un < n_units;
    Unit nxt = cur;
    if (has_next) nxt = unit_at(un);

    bf16x8 qf[KSTEPS];
    u32x4 pv[NCP];
    float m_run[NH];  // running max per head, log2 units (raw score x scale_log2)
    float l_run[NH];
#pragma unroll
    for (int p = 0; p < NH; ++p) {
      m_run[p] = -INFINITY;
      l_run[p] = 0.0f;
    }
    f32x16 o[DT];  // tile dt belongs to head dt (PAIR) or to the one head
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[dt][r] = 0.0f;

    for (int kb = 0; kb < nkb; ++kb) {
      // Everything this wave issued before is done: the current block (and,
      // at a unit's first block, its Q), and the stores of the unit before.
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      if (kb == 0) {
#pragma unroll
        for (int kk = 0; kk < KSTEPS; ++kk)
          qf[kk] = __builtin_bit_cast(bf16x8, sQ[swz<CPR>(col, kk * 2 + half)]);
        if (pending) {
#pragma unroll
          for (int j = 0; j < NCP; ++j) pv[j] = sK[b ^ 1][j * 64 + lane];
        }
        // sQ and the other buffer are read out: they can be refilled.
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      }
      // Prefetch the wave's next block into the other buffer: the next key
      // block of this unit, or the next unit's Q and first key block.
      if (kb + 1 < nkb) {
        copy_block(cur.base + D, (kb + 1) * 32, cur.L, lk + (b ^ 1) * BUF);
        copy_block(cur.base + 2 * D, (kb + 1) * 32, cur.L, lv + (b ^ 1) * BUF);
      } else if (has_next) {
        copy_block(nxt.base, nxt.q0, nxt.L, lq);
        copy_block(nxt.base + D, 0, nxt.L, lk + (b ^ 1) * BUF);
        copy_block(nxt.base + 2 * D, 0, nxt.L, lv + (b ^ 1) * BUF);
      }
      if (kb == 0 && pending) {
#pragma unroll
        for (int j = 0; j < NCP; ++j) {
          const int row = j * RPC + crow;
          if (row < p_rows)
            __builtin_nontemporal_store(
                pv[j], reinterpret_cast<u32x4*>(p_ob + (size_t)row * D + copy_chunk<CPR>(lane, j) * 8));
        }
        pending = false;
      }
      const int k0 = kb * 32;
      const u32x4* kbuf = sK[b];
      const u32x4* vbuf = sV[b];

      // S^T block of each head: rows = keys k0..k0+31 (A operand = K),
      // cols = queries; head p is steps p*KS .. p*KS+KS-1 of the row slice.
      f32x16 s[NH];
#pragma unroll
      for (int p = 0; p < NH; ++p) {
#pragma unroll
        for (int r = 0; r < 16; ++r) s[p][r] = 0.0f;
#pragma unroll
        for (int kk = p * KS; kk < (p + 1) * KS; ++kk)
          s[p] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8, kbuf[swz<CPR>(col, kk * 2 + half)]), qf[kk], s[p], 0, 0, 0);
      }

      // Register r holds the score of key k0 + 8*(r/4) + 4*half + r%4; only
      // the text's last block has keys past its end (uniform branch).
      if (k0 + 32 > cur.L) {
#pragma unroll
        for (int p = 0; p < NH; ++p)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (k0 + 8 * (r >> 2) + 4 * half + (r & 3) >= cur.L) s[p][r] = -INFINITY;
      }
      float alpha[NH];
#pragma unroll
      for (int p = 0; p < NH; ++p) {
        float mloc = s[p][0];
#pragma unroll
        for (int r = 1; r < 16; ++r) mloc = fmaxf(mloc, s[p][r]);
        mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
        const float m_new = fmaxf(m_run[p], mloc * scale_log2);
        float psum = 0.0f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          s[p][r] = __builtin_amdgcn_exp2f(fmaf(s[p][r], scale_log2, -m_new));
          psum += s[p][r];
        }
        psum += __shfl_xor(psum, 32, 64);
        if (kb == 0) {
          l_run[p] = psum;  // o is still zero: nothing to rescale
        } else {
          alpha[p] = __builtin_amdgcn_exp2f(m_run[p] - m_new);
          l_run[p] = fmaf(l_run[p], alpha[p], psum);
        }
        m_run[p] = m_new;
      }
      if (kb > 0) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[dt][r] *= alpha[PAIR ? dt : 0];
      }

      // O^T += V^T P^T over two 16-key halves c: slot j of this lane is key
      // 16c + 8*(j/4) + 4*half + j%4, the same key for the P (B) and V (A)
      // operands.
      bf16x8 pb[NH][2];
#pragma unroll
      for (int p = 0; p < NH; ++p)
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int j = 0; j < 8; ++j) pb[p][c][j] = (__bf16)s[p][8 * c + j];
      const char* vbytes = reinterpret_cast<const char*>(vbuf);
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
          o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[PAIR ? dt : 0][c], o[dt], 0, 0, 0);
        }
      }
      b ^= 1;
    }

    // O^T register r of tile dt: head feature dt*32 + 8*(r/4) + 4*half + r%4
    // of query q0 + col.  Stage the normalised bf16 block in the K buffer of
    // the unit's last key block (row = query; its K reads went into MFMAs).
    float inv[NH];
#pragma unroll
    for (int p = 0; p < NH; ++p) inv[p] = 1.0f / l_run[p];
    char* obytes = reinterpret_cast<char*>(sK[b ^ 1]);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const float inv_h = inv[PAIR ? dt : 0];
        uint2 w;
        w.x = pack_bf16x2(o[dt][4 * g + 0] * inv_h, o[dt][4 * g + 1] * inv_h);
        w.y = pack_bf16x2(o[dt][4 * g + 2] * inv_h, o[dt][4 * g + 3] * inv_h);
        *reinterpret_cast<uint2*>(obytes + swz<CPR>(col, dt * 4 + g) * 16 + half * 8) = w;
      }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    p_ob = out + (size_t)(cur.beg + cur.q0) * D + (size_t)cur.h * DH;
    p_rows = cur.L - cur.q0;
    if (!has_next) {
      // Last unit of this wave: store now.
#pragma unroll
      for (int j = 0; j < NCP; ++j) {
        const int row = j * RPC + crow;
        const u32x4 v = sK[b ^ 1][j * 64 + lane];
        if (row < p_rows)
          __builtin_nontemporal_store(
              v, reinterpret_cast<u32x4*>(p_ob + (size_t)row * D + copy_chunk<CPR>(lane, j) * 8));
      }
      break;
    }
    // The next unit's first block stores this one after its data arrived.
    pending = true;
    cur = nxt;
    u = un;
  }
}

}  // namespace

hipError_t launch_attention(const uint16_t* qkv, uint16_t* out, const int32_t* cu,
                            const uint32_t* items, int n_items, int n_heads, int d_head,
                            hipStream_t stream) {
  if (n_items <= 0) return hipSuccess;
  if (d_head != 64 && (d_head != 32 || n_heads % 2)) return hipErrorInvalidValue;
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)d_head);
  // 32-dimensional heads go in adjacent pairs: one 64-wide row slice each.
  const int slices = d_head == 64 ? n_heads : n_heads / 2;
  const int n_units = n_items * slices;
  const dim3 grid((unsigned)((n_units + UNITS_PER_WAVE - 1) / UNITS_PER_WAVE));
  if (d_head == 64)
    hipLaunchKernelGGL((attention_varlen_kernel<64, false>), grid, dim3(64), 0, stream, qkv, out, cu,
                       items, slices, scale_log2, n_units);
  else
    hipLaunchKernelGGL((attention_varlen_kernel<64, true>), grid, dim3(64), 0, stream, qkv, out, cu,
                       items, slices, scale_log2, n_units);
  return hipGetLastError();
}

int row_block_items(const int64_t* cu, int64_t n_texts, uint32_t* items) {
  // (text, 32-row block) pairs, longest text first; ties keep text order.
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
