// Token-major linear layers on bf16 MFMA (gfx950): Y = epi(X W^T + b).
//
// X is the packed token matrix [M, K] (M = tokens of the chunk, no padding),
// W the layer weight repacked to [N, K] so both operands are K-contiguous.
//
// Tiling.  A workgroup computes a BM x BN tile of Y (tokens x features) with
// WAVES_M x WAVES_N waves; each wave owns a (BM/WAVES_M) x (BN/WAVES_N)
// sub-tile held as 32 x 32 v_mfma_f32_32x32x16_bf16 accumulators.  K is
// walked in BK-wide stages (64 or 32) through a double-buffered LDS tile.
//
// Staging.  Stage k+1 is copied straight from global memory into the idle
// LDS buffer (global_load_lds_dwordx4, 1 KB per wave instruction) while
// stage k runs on the MFMA units; one wait and one barrier per stage.  An
// LDS row holds BK bf16 of one X or W row as CPR = BK/8 16-byte chunks; the
// logical chunk c of row r is stored at position c ^ f(r), with
//   CPR = 8: f(r) = (r & 7) ^ ((r >> 3) & 1),
//   CPR = 4: f(r) = ((r >> 1) & 3) ^ ((r >> 3) & 1).
// A fragment read takes one logical chunk from 32 consecutive rows; with
// either f, any 8 aligned rows fall on 8 different 16-byte slots of a
// 128-byte window and any 16 aligned rows on 16 different slots of a
// 256-byte window, so the reads are free of bank conflicts whether the LDS
// serves a 16-byte read 8 lanes at a time over 32 banks or 16 lanes at a
// time over 64 banks.  A copy instruction writes 64 consecutive slots, so
// each lane fetches the logical chunk that belongs in its slot.
//
// Occupancy.  Every configuration runs 2 waves per SIMD.  8-wave 256 x 256
// tiles take the whole CU (128 KB of LDS); 4-wave tiles with BK = 32 need
// at most 64 KB, so two workgroups share a CU and one's epilogue overlaps
// the other's MFMA loop.
//
// Operand roles.  The MFMA A operand is the weight tile and B the token
// tile, so the accumulators hold Y^T: each lane owns one token row and four
// consecutive features per register group, which makes the epilogue (bias,
// GELU, residual, bf16 store) 8-byte vector accesses.
//
// Every output row is computed from its own input row with a fixed K order
// (no split-K, no atomics), so a text's result does not depend on which
// other texts share its SuperBatch or chunk, nor on the tile configuration.
#include "device_common.h"
#include "kernels.h"

namespace surge {
namespace {

constexpr int STATS_WIDTH = 64;  // features per row-statistics partial

// Wait until at most `later` stages' copies (CPS instructions each) issued
// after the one needed next are still in flight.  The vector memory counter
// retires a wave's loads in issue order.
template <int CPS>
__device__ __forceinline__ void wait_copies(int later) {
  if (later <= 0)
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else if (later == 1)
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(CPS) : "memory");
  else
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * CPS) : "memory");
}

// Tile order.  Workgroups are dispatched round-robin over the 8 XCDs
// (block b runs on XCD b % 8), each with its own 4 MB L2, so the order in
// which one XCD walks its tiles decides what its L2 can reuse.
//   ORDER_ROW_GROUPS: each XCD walks a contiguous eighth of the tile grid in
//     groups of 8 token-row blocks, feature tile outer: a weight tile is
//     reused by 8 row blocks and 8 X row blocks stay resident meanwhile.
//   ORDER_FEATURE_HALVES: the XCDs form 2 feature halves x 4 token-row
//     quarters and each walks its rectangle as above, so an XCD touches half
//     of W (FFN1's 4.7 MB W does not fit one L2, half of it does).  Falls
//     back to ORDER_ROW_GROUPS when the rectangles do not divide evenly.
// The blocks beyond the last full eighth keep their own index.
constexpr int ORDER_ROW_GROUPS = 0;
constexpr int ORDER_FEATURE_HALVES = 1;

template <int ORDER>
__device__ __forceinline__ void tile_coords(int b, int n_tiles, int tiles_n, int* tm, int* tn) {
  const int tiles_m = n_tiles / tiles_n;
  const int xcd = b & 7;
  const int local = b >> 3;
  int t, m_base = 0, n_base = 0, m_cnt = tiles_m, n_cnt = tiles_n;
  if (ORDER == ORDER_FEATURE_HALVES && tiles_n % 2 == 0 && tiles_m % 4 == 0) {
    n_cnt = tiles_n / 2;
    m_cnt = tiles_m / 4;
    n_base = (xcd & 1) * n_cnt;
    m_base = (xcd >> 1) * m_cnt;
    t = local;
  } else {
    const int per_xcd = n_tiles >> 3;
    t = b < (per_xcd << 3) ? xcd * per_xcd + local : b;
  }
  const int grp = t / (8 * n_cnt);
  const int in = t - grp * 8 * n_cnt;
  const int rows = min(8, m_cnt - grp * 8);
  *tn = n_base + in / rows;
  *tm = m_base + grp * 8 + in % rows;
}


template <int BM, int BN, int BK, int NBUF, int WAVES_M, int WAVES_N, int EPI, int ORDER>
__global__ __launch_bounds__(WAVES_M* WAVES_N * 64) __attribute__((amdgpu_waves_per_eu(2)))
void linear_bf16_kernel(const uint16_t* __restrict__ X, const uint16_t* __restrict__ W,
                        const float* __restrict__ bias, const uint16_t* __restrict__ R,
                        uint16_t* __restrict__ Y, int M, int N, int K, int tiles_n, int n_tiles,
                        LinearExtra ex) {
  constexpr int NWAVES = WAVES_M * WAVES_N;
  constexpr int WM = BM / WAVES_M;  // tokens per wave
  constexpr int WN = BN / WAVES_N;  // features per wave
  constexpr int TM = WM / 32;       // 32-token accumulator tiles per wave
  constexpr int TN = WN / 32;       // 32-feature accumulator tiles per wave
  constexpr int NT = NWAVES * 64;
  constexpr int CPR = BK / 8;       // 16-byte chunks per LDS row
  constexpr int RPC = 64 / CPR;     // rows one wave copy instruction fills
  constexpr int XI = BM / (RPC * NWAVES);  // copy instructions per wave per stage, X tile
  constexpr int WI = BN / (RPC * NWAVES);  // ... W tile
  static_assert(XI * RPC * NWAVES == BM && WI * RPC * NWAVES == BN, "tile/wave mismatch");
  static_assert(CPR == 4 || NWAVES % 2 == 0, "copy slot phase needs an even wave count");
  static_assert(NBUF >= 2 && NBUF <= 4, "2 to 4 LDS stage buffers");
  static_assert((XI + WI) * (NBUF - 2) < 64, "copies in flight must fit the counter");

  // Main loop: NBUF stage buffers; buffer b holds X rows at
  // smem[b*SSTAGE ..] and W rows after them.  Epilogue: the same memory
  // holds the bf16 output tile.
  constexpr int SSTAGE = (BM + BN) * CPR;
  constexpr int SMEM = NBUF * SSTAGE > BM * BN / 8 ? NBUF * SSTAGE : BM * BN / 8;
  __shared__ u32x4 smem[SMEM];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;

  int tn, tm;
  tile_coords<ORDER>(blockIdx.x, n_tiles, tiles_n, &tm, &tn);
  const int m0 = tm * BM;
  const int n0 = tn * BN;
  const int wn0 = (wave % WAVES_N) * WN;
  const int wm0 = (wave / WAVES_N) * WM;

  // LayerNorm factors of this lane's rows (fused LayerNorm epilogues),
  // fetched now so their latency hides behind the main loop.
  float2 rowf[TM];
#pragma unroll
  for (int j = 0; j < TM; ++j) {
    rowf[j] = make_float2(0.0f, 0.0f);
    if constexpr (EPI == EPI_FOLD || EPI == EPI_FOLD_GELU || EPI == EPI_LNRES_STATS)
      rowf[j] = ex.rows_in[min(m0 + wm0 + j * 32 + (lane & 31), M - 1)];
  }

  f32x16 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nkt = K / BK;
  const int l32 = lane & 31;
  const int lhi = lane >> 5;

  // Lane l of wave w, copy j, fills LDS slot p = (j*NWAVES + w)*64 + l of a
  // tile: row p / CPR, stored chunk l % CPR.  Its logical chunk
  // (l % CPR) ^ f(row) is the same for every j:
  //   CPR = 8: (l & 7) ^ (l >> 3) ^ (w & 1)   (NWAVES even),
  //   CPR = 4: (l & 3) ^ ((l >> 3) & 3) ^ (l >> 5).
  // Its rows are NWAVES * RPC apart.
  constexpr int DSTEP = NWAVES * RPC;
  const int drow = wave * RPC + lane / CPR;
  const int dch = copy_chunk<CPR>(lane, wave);
  const uint16_t* xg[XI];
#pragma unroll
  for (int j = 0; j < XI; ++j)
    xg[j] = X + (size_t)min(m0 + drow + j * DSTEP, M - 1) * K + dch * 8;  // rows past M: clamped, never stored
  const uint16_t* wg = W + (size_t)(n0 + drow) * K + dch * 8;
  const size_t wgstep = (size_t)DSTEP * K;
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_address(smem) + wave * 64 * 16);
  constexpr uint32_t STAGE_BYTES = SSTAGE * 16;
  constexpr uint32_t COPY_BYTES = NWAVES * 64 * 16;

#define SURGE_ISSUE_STAGE(kk_, b_)                                                        \
  do {                                                                                    \
    const int ko_ = (kk_) * BK;                                                           \
    const uint32_t base_ = lds0 + (uint32_t)(b_) * STAGE_BYTES;                           \
    _Pragma("unroll") for (int j = 0; j < XI; ++j)                                        \
      copy_to_lds16(xg[j] + ko_, base_ + j * COPY_BYTES);                                 \
    _Pragma("unroll") for (int j = 0; j < WI; ++j)                                        \
      copy_to_lds16(wg + j * wgstep + ko_, base_ + BM * CPR * 16 + j * COPY_BYTES);       \
  } while (0)

  // Prologue: stages 0 .. NBUF-1 in flight; wait for stage 0, publish it
  // and read its first fragments.
#pragma unroll
  for (int st = 0; st < NBUF; ++st)
    if (st < nkt) SURGE_ISSUE_STAGE(st, st);
  wait_copies<XI + WI>(min(NBUF - 1, nkt - 1));
  __syncthreads();
  constexpr int S = BK / 16;   // 16-wide MFMA steps per stage
  constexpr int NR = TN + TM;  // fragment reads per step
  constexpr int NM = TN * TM;  // MFMAs per step
  static_assert(S % 2 == 0, "fragment parity must restart at every stage");
  static_assert(NM >= NR, "interleave needs at least one MFMA per read");
  bf16x8 fa[2][TN], fb[2][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
    fa[0][i] = __builtin_bit_cast(bf16x8, smem[BM * CPR + swz<CPR>(wn0 + i * 32 + l32, lhi)]);
#pragma unroll
  for (int j = 0; j < TM; ++j)
    fb[0][j] = __builtin_bit_cast(bf16x8, smem[swz<CPR>(wm0 + j * 32 + l32, lhi)]);

  // One stage per trip.  Steps 0 .. S-2 run their MFMAs with the fragment
  // reads of the following step interleaved one by one (pinned with
  // scheduling group barriers).  Then the wave waits for its copies of
  // stage k+1 and all waves meet: stage k+1 is published and nobody reads
  // stage k's buffer any more, so the copies of stage k+NBUF go into it.
  // The last step's MFMAs, which need no LDS, run after the barrier while
  // the first fragments of stage k+1 are read, so the MFMA pipe does not
  // wait for LDS at the stage boundary.  (On the last trip those reads hit
  // a stale buffer and are discarded.)
  int cur_buf = 0;
  for (int kt = 0; kt < nkt; ++kt) {
    const u32x4* sx = smem + cur_buf * SSTAGE;
    const u32x4* sw = sx + BM * CPR;
#pragma unroll
    for (int ks = 0; ks + 1 < S; ++ks) {
      const int cur = ks & 1;
      const int ch = (ks + 1) * 2 + lhi;
#pragma unroll
      for (int i = 0; i < TN; ++i)
        fa[cur ^ 1][i] = __builtin_bit_cast(bf16x8, sw[swz<CPR>(wn0 + i * 32 + l32, ch)]);
#pragma unroll
      for (int j = 0; j < TM; ++j)
        fb[cur ^ 1][j] = __builtin_bit_cast(bf16x8, sx[swz<CPR>(wm0 + j * 32 + l32, ch)]);
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[cur][i], fb[cur][j], acc[i][j], 0,
                                                              0, 0);
    }
#pragma unroll
    for (int ks = 0; ks + 1 < S; ++ks) {
#pragma unroll
      for (int t = 0; t < NR; ++t) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
      }
      __builtin_amdgcn_sched_group_barrier(0x008, NM - NR, 0);
    }
    // stages issued after stage kt+1: up to kt + NBUF - 1, capped at the end
    wait_copies<XI + WI>(min(kt + NBUF - 1, nkt - 1) - (kt + 1));
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // this stage's reads are done
    __syncthreads();
    if (kt + NBUF < nkt) SURGE_ISSUE_STAGE(kt + NBUF, cur_buf);
    cur_buf = cur_buf + 1 == NBUF ? 0 : cur_buf + 1;
    const u32x4* nx = smem + cur_buf * SSTAGE;
    const u32x4* nw = nx + BM * CPR;
#pragma unroll
    for (int i = 0; i < TN; ++i)
      fa[0][i] = __builtin_bit_cast(bf16x8, nw[swz<CPR>(wn0 + i * 32 + l32, lhi)]);
#pragma unroll
    for (int j = 0; j < TM; ++j)
      fb[0][j] = __builtin_bit_cast(bf16x8, nx[swz<CPR>(wm0 + j * 32 + l32, lhi)]);
#pragma unroll
    for (int i = 0; i < TN; ++i)
#pragma unroll
      for (int j = 0; j < TM; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[1][i], fb[1][j], acc[i][j], 0, 0, 0);
#pragma unroll
    for (int t = 0; t < NR; ++t) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, NM - NR, 0);
  }
#undef SURGE_ISSUE_STAGE

  // Epilogue, staged through LDS so global traffic is whole rows.
  // acc[i][j] register r holds Y[m][n] with
  //   m = m0 + wm0 + j*32 + lane%32
  //   n = n0 + wn0 + i*32 + 8*(r/4) + 4*(lane/32) + r%4,
  // i.e. registers 4g..4g+3 are the 8-byte output unit
  // (wn0 + i*32 + 8g)/4 + lane/32 of row m (a row holds BN/4 such units).
  // The LDS holds the BM x BN tile as bf16 rows of BN/4 8-byte units; unit
  // u of row r sits at u ^ (r & 31), so the 32 rows an accumulator register
  // spans fall on distinct banks and a 16-byte pair {2k, 2k+1} stays
  // together (possibly with its halves swapped).
  //   1. (residual modes) every thread copies whole rows of R into the tile
  //      with 16-byte coalesced loads, all issued before any is used;
  //   2. each lane finishes its accumulators (bias or folded LayerNorm,
  //      GELU, residual read back from the tile), rounds once to bf16 and
  //      writes the tile; the statistics modes also sum the rounded values
  //      of each of its rows;
  //   3. every thread stores whole rows of the tile with 16-byte stores.
  {
    constexpr bool FOLD = EPI == EPI_FOLD || EPI == EPI_FOLD_GELU;
    constexpr bool GELU = EPI == EPI_BIAS_GELU || EPI == EPI_FOLD_GELU;
    constexpr bool RES = EPI == EPI_BIAS_RESIDUAL || EPI == EPI_RES_STATS || EPI == EPI_LNRES_STATS;
    constexpr bool LNRES = EPI == EPI_LNRES_STATS;
    constexpr bool STATS = EPI == EPI_RES_STATS || EPI == EPI_LNRES_STATS;
    constexpr int U = BN / 4;            // 8-byte units per row
    constexpr int PAIRS = BN / 8;        // 16-byte pairs per row
    constexpr int RPI = NT / PAIRS;      // rows per coalesced iteration
    constexpr int ITER = BM / RPI;
    static_assert(BM % RPI == 0 && U >= 32, "epilogue shape");
    uint2* t8 = reinterpret_cast<uint2*>(smem);
    u32x4* t16 = smem;
    const int cp = threadIdx.x % PAIRS;  // this thread's 16-byte pair in a row
    const int cr = threadIdx.x / PAIRS;

    // Per-row LayerNorm factors (rstd, -mean rstd) of the folded input
    // (FOLD: X's rows) or of the residual (LNRES: R's rows), loaded before
    // the main loop.
    float rs[TM], nm[TM];
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      rs[j] = rowf[j].x;
      nm[j] = rowf[j].y;
    }

    if constexpr (RES) {
      u32x4 rv[ITER];
#pragma unroll
      for (int it = 0; it < ITER; ++it) {
        const int m = min(m0 + it * RPI + cr, M - 1);
        rv[it] = *reinterpret_cast<const u32x4*>(R + (size_t)m * N + n0 + 8 * cp);
      }
#pragma unroll
      for (int it = 0; it < ITER; ++it) {
        const int r = it * RPI + cr;
        const int ph = (2 * cp) ^ (r & 31);  // physical unit of logical unit 2cp
        u32x4 v = rv[it];
        if (ph & 1) v = u32x4{v[2], v[3], v[0], v[1]};
        t16[r * PAIRS + (ph >> 1)] = v;
      }
      __syncthreads();
    }
    // Statistics partials are 64 features wide in every tile configuration
    // (two 32-feature accumulator tiles, summed in the same order), so a
    // row's statistics do not depend on the tile shape of its chunk.
    constexpr int PW = STATS_WIDTH;
    constexpr int NPW = WN / PW;  // partials per wave
    static_assert(WN % PW == 0 && PW % 32 == 0, "statistics partial shape");
    float st_s[TM][NPW], st_q[TM][NPW];
#pragma unroll
    for (int j = 0; j < TM; ++j)
#pragma unroll
      for (int q = 0; q < NPW; ++q) st_s[j][q] = st_q[j][q] = 0.0f;
#pragma unroll
    for (int i = 0; i < TN; ++i) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int u = (wn0 + i * 32 + 8 * g) / 4 + lhi;
        const float4 bb = *reinterpret_cast<const float4*>(bias + n0 + 4 * u);
        float4 cs = {0.0f, 0.0f, 0.0f, 0.0f}, gg = cs, be = cs;
        if constexpr (FOLD) cs = *reinterpret_cast<const float4*>(ex.col_s + n0 + 4 * u);
        if constexpr (LNRES) {
          gg = *reinterpret_cast<const float4*>(ex.gamma + n0 + 4 * u);
          be = *reinterpret_cast<const float4*>(ex.beta + n0 + 4 * u);
        }
#pragma unroll
        for (int j = 0; j < TM; ++j) {
          const int r = wm0 + j * 32 + l32;
          float o0, o1, o2, o3;
          if constexpr (FOLD) {
            o0 = fmaf(rs[j], acc[i][j][4 * g + 0], fmaf(nm[j], cs.x, bb.x));
            o1 = fmaf(rs[j], acc[i][j][4 * g + 1], fmaf(nm[j], cs.y, bb.y));
            o2 = fmaf(rs[j], acc[i][j][4 * g + 2], fmaf(nm[j], cs.z, bb.z));
            o3 = fmaf(rs[j], acc[i][j][4 * g + 3], fmaf(nm[j], cs.w, bb.w));
          } else {
            o0 = acc[i][j][4 * g + 0] + bb.x;
            o1 = acc[i][j][4 * g + 1] + bb.y;
            o2 = acc[i][j][4 * g + 2] + bb.z;
            o3 = acc[i][j][4 * g + 3] + bb.w;
          }
          if constexpr (GELU) {
            o0 = gelu_erf(o0);
            o1 = gelu_erf(o1);
            o2 = gelu_erf(o2);
            o3 = gelu_erf(o3);
          }
          uint2& cell = t8[r * U + (u ^ (r & 31))];
          if constexpr (RES) {
            const uint2 rr = cell;
            float r0 = __uint_as_float(rr.x << 16);
            float r1 = __uint_as_float(rr.x & 0xffff0000u);
            float r2 = __uint_as_float(rr.y << 16);
            float r3 = __uint_as_float(rr.y & 0xffff0000u);
            if constexpr (LNRES) {
              r0 = fmaf(fmaf(r0, rs[j], nm[j]), gg.x, be.x);
              r1 = fmaf(fmaf(r1, rs[j], nm[j]), gg.y, be.y);
              r2 = fmaf(fmaf(r2, rs[j], nm[j]), gg.z, be.z);
              r3 = fmaf(fmaf(r3, rs[j], nm[j]), gg.w, be.w);
            }
            o0 += r0;
            o1 += r1;
            o2 += r2;
            o3 += r3;
          }
          uint2 out;
          out.x = pack_bf16x2(o0, o1);
          out.y = pack_bf16x2(o2, o3);
          cell = out;
          if constexpr (STATS) {
            const float v0 = __uint_as_float(out.x << 16), v1 = __uint_as_float(out.x & 0xffff0000u);
            const float v2 = __uint_as_float(out.y << 16), v3 = __uint_as_float(out.y & 0xffff0000u);
            const int q = i / (PW / 32);
            st_s[j][q] += (v0 + v1) + (v2 + v3);
            st_q[j][q] = fmaf(v0, v0, fmaf(v1, v1, fmaf(v2, v2, fmaf(v3, v3, st_q[j][q]))));
          }
        }
      }
    }
    if constexpr (STATS) {
      // The lane and its partner (lane ^ 32) hold complementary halves of
      // each PW-feature slice; partial index = first feature / PW.
      const int part0 = (n0 + wn0) / PW;
      constexpr float inv_w = 1.0f / (float)PW;
#pragma unroll
      for (int j = 0; j < TM; ++j) {
        const int m = m0 + wm0 + j * 32 + l32;
#pragma unroll
        for (int q = 0; q < NPW; ++q) {
          const float s1 = st_s[j][q] + __shfl_xor(st_s[j][q], 32, 64);
          const float q1 = st_q[j][q] + __shfl_xor(st_q[j][q], 32, 64);
          if (lhi == 0 && m < M) {
            const float mean = s1 * inv_w;
            ex.stats_out[(size_t)(part0 + q) * M + m] =
                make_float2(mean, fmaxf(q1 * inv_w - mean * mean, 0.0f));
          }
        }
      }
    }
    __syncthreads();
    u32x4 ov[ITER];
#pragma unroll
    for (int it = 0; it < ITER; ++it) {
      const int r = it * RPI + cr;
      const int ph = (2 * cp) ^ (r & 31);
      ov[it] = t16[r * PAIRS + (ph >> 1)];
      if (ph & 1) ov[it] = u32x4{ov[it][2], ov[it][3], ov[it][0], ov[it][1]};
    }
#pragma unroll
    for (int it = 0; it < ITER; ++it) {
      const int m = m0 + it * RPI + cr;
      if (m < M) *reinterpret_cast<u32x4*>(Y + (size_t)m * N + n0 + 8 * cp) = ov[it];
    }
  }
}

template <int BM, int BN, int BK, int NBUF, int WAVES_M, int WAVES_N>
hipError_t launch_tiles(const uint16_t* X, const uint16_t* W, const float* bias, const uint16_t* R,
                        uint16_t* Y, int64_t M, int N, int K, int epi, const LinearExtra& ex,
                        hipStream_t stream) {
  const int tiles_n = N / BN;
  const int64_t tiles_m = (M + BM - 1) / BM;
  const int n_tiles = (int)(tiles_m * tiles_n);
  const dim3 grid((unsigned)n_tiles);
  const dim3 block(WAVES_M * WAVES_N * 64);
#define SURGE_LAUNCH_EPI(E, O)                                                                \
  hipLaunchKernelGGL((linear_bf16_kernel<BM, BN, BK, NBUF, WAVES_M, WAVES_N, E, O>), grid, block, \
                     0, stream, X, W, bias, R, Y, (int)M, N, K, tiles_n, n_tiles, ex)
  switch (epi) {
    case EPI_BIAS: SURGE_LAUNCH_EPI(EPI_BIAS, ORDER_ROW_GROUPS); break;
    case EPI_BIAS_GELU: SURGE_LAUNCH_EPI(EPI_BIAS_GELU, ORDER_FEATURE_HALVES); break;
    case EPI_BIAS_RESIDUAL: SURGE_LAUNCH_EPI(EPI_BIAS_RESIDUAL, ORDER_ROW_GROUPS); break;
    case EPI_FOLD: SURGE_LAUNCH_EPI(EPI_FOLD, ORDER_ROW_GROUPS); break;
    case EPI_FOLD_GELU: SURGE_LAUNCH_EPI(EPI_FOLD_GELU, ORDER_FEATURE_HALVES); break;
    case EPI_RES_STATS: SURGE_LAUNCH_EPI(EPI_RES_STATS, ORDER_ROW_GROUPS); break;
    default: SURGE_LAUNCH_EPI(EPI_LNRES_STATS, ORDER_ROW_GROUPS); break;
  }
#undef SURGE_LAUNCH_EPI
  return hipGetLastError();
}

}  // namespace

// The tile configuration of an [M, N] output: 256 x 256 tiles (8 waves of
// 64 tokens x 128 features) where the feature count allows it and there are
// enough token rows to fill the chip; 128 x 128 tiles (4 waves of 64 x 64)
// otherwise.
static bool big_tiles(int64_t M, int N) { return N % 256 == 0 && M >= 8192; }

int linear_stats_width(int64_t, int) { return STATS_WIDTH; }

hipError_t launch_linear(const uint16_t* X, const uint16_t* W, const float* bias, const uint16_t* R,
                         uint16_t* Y, int64_t M, int N, int K, int epi, const LinearExtra& ex,
                         hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  if (big_tiles(M, N))
    return launch_tiles<256, 256, 64, 2, 4, 2>(X, W, bias, R, Y, M, N, K, epi, ex, stream);
  return launch_tiles<128, 128, 64, 2, 2, 2>(X, W, bias, R, Y, M, N, K, epi, ex, stream);
}

}  // namespace surge
