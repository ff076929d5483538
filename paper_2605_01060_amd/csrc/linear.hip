// Token-major linear layers on bf16 MFMA (gfx950): Y = epi(X W^T + b).
//
// X is the packed token matrix [M, K] (M = tokens of the chunk, no padding),
// W the layer weight repacked to [N, K] so both operands are K-contiguous.
//
// Tiling.  A workgroup computes BM x BN tiles of Y (tokens x features) with
// WAVES_M x WAVES_N waves; each wave owns a (BM/WAVES_M) x (BN/WAVES_N)
// sub-tile held as 32 x 32 v_mfma_f32_32x32x16_bf16 accumulators.  K is
// walked in 64-wide stages through a double-buffered LDS tile.
//
// Persistence.  The grid holds as many workgroups as fit on the chip at
// once; workgroup b computes tiles b, b + G, b + 2G, ... (G = grid size).
// The copy pipeline runs on across tile boundaries: the next tile's first
// stage is copied while the current tile's last stage is on the MFMA units,
// and its second stage as soon as each wave has finished its epilogue.  A
// tile therefore never starts on an empty pipeline, and no workgroup launch
// separates two tiles.
//
// Epilogue memory.  The buffer released by a tile's last stage is idle
// until the next tile's second stage is copied into it, so each wave uses
// the slots its own copies of that stage will fill as its 4 KB epilogue
// region, and issues those copies when its epilogue is done (no other wave
// touches the slots, so no barrier is needed).  The tile's per-feature
// vectors (bias, and the LayerNorm columns of the fused forms) are copied
// into LDS once per tile at its start, so the epilogue reads them from LDS
// instead of every lane fetching them again from global memory.  The
// output rows and the residual rows are touched once per launch, so they
// are stored and loaded nontemporally, leaving the L2 to the operand tiles
// that other workgroups read again.
//
// Staging.  Stage k+2 is copied straight from global memory into the LDS
// buffer stage k has just released (global_load_lds_dwordx4, 1 KB per wave
// instruction) while stage k+1 runs on the MFMA units; one wait and one
// barrier per stage.  An LDS row holds 64 bf16 of one X or W row as eight
// 16-byte chunks; the logical chunk c of row r is stored at position
// c ^ (r & 7) ^ ((r >> 3) & 1).  A fragment read takes one logical chunk
// from 32 consecutive rows; any 8 aligned rows fall on 8 different 16-byte
// slots of a 128-byte window and any 16 aligned rows on 16 different slots
// of a 256-byte window, so the reads are free of bank conflicts whether the
// LDS serves a 16-byte read 8 lanes at a time over 32 banks or 16 lanes at
// a time over 64 banks.  A copy instruction writes 64 consecutive slots, so
// each lane fetches the logical chunk that belongs in its slot.
//
// Occupancy.  Both configurations run 2 waves per SIMD: an 8-wave
// 256 x 256 workgroup takes 128 KB of stage buffers plus at most 6 KB of
// per-feature vectors (one per CU); a 4-wave 128 x 128 workgroup takes
// 64 + 3 KB (two per CU).
//
// Operand roles.  The MFMA A operand is the weight tile and B the token
// tile, so the accumulators hold Y^T: each lane owns one token row and four
// consecutive features per register group.
//
// Every output row is computed from its own input row with a fixed K order
// (no split-K, no atomics), so a text's result does not depend on which
// other texts share its SuperBatch or chunk, nor on the tile configuration.
#include <algorithm>

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

// Epilogue region layout: 32 rows x 64 bf16, a row as 16 8-byte units;
// unit u of row r sits at u ^ rsw(r).  The 32 rows that one 8-byte access
// of a wave spans (one unit each) land on distinct banks under either LDS
// bank geometry, and an aligned 16-byte pair {2k, 2k+1} stays together
// (halves swapped when rsw(r) is odd).
__device__ __forceinline__ int rsw(int r) { return (r & 15) ^ ((r >> 4) & 1); }

// Finishes four consecutive features of one output row and rounds them to
// bf16: bias (or the folded LayerNorm rs * a + (nm * s + b)), GELU, then
// the residual `res` (LayerNorm-applied as (r rs + nm) g + beta in the
// LNRES mode).
template <int EPI>
__device__ __forceinline__ uint2 finish4(const float (&a)[4], float4 bb, float4 cs, float4 gg,
                                         float4 be, float rs, float nm, uint2 res) {
  constexpr bool FOLD = EPI == EPI_FOLD || EPI == EPI_FOLD_GELU;
  constexpr bool GELU = EPI == EPI_BIAS_GELU || EPI == EPI_FOLD_GELU;
  constexpr bool RES = EPI == EPI_BIAS_RESIDUAL || EPI == EPI_RES_STATS || EPI == EPI_LNRES_STATS;
  constexpr bool LNRES = EPI == EPI_LNRES_STATS;
  float o0, o1, o2, o3;
  if constexpr (FOLD) {
    o0 = fmaf(rs, a[0], fmaf(nm, cs.x, bb.x));
    o1 = fmaf(rs, a[1], fmaf(nm, cs.y, bb.y));
    o2 = fmaf(rs, a[2], fmaf(nm, cs.z, bb.z));
    o3 = fmaf(rs, a[3], fmaf(nm, cs.w, bb.w));
  } else {
    o0 = a[0] + bb.x;
    o1 = a[1] + bb.y;
    o2 = a[2] + bb.z;
    o3 = a[3] + bb.w;
  }
  if constexpr (GELU) {
    o0 = gelu_erf(o0);
    o1 = gelu_erf(o1);
    o2 = gelu_erf(o2);
    o3 = gelu_erf(o3);
  }
  if constexpr (RES) {
    float r0 = __uint_as_float(res.x << 16);
    float r1 = __uint_as_float(res.x & 0xffff0000u);
    float r2 = __uint_as_float(res.y << 16);
    float r3 = __uint_as_float(res.y & 0xffff0000u);
    if constexpr (LNRES) {
      r0 = fmaf(fmaf(r0, rs, nm), gg.x, be.x);
      r1 = fmaf(fmaf(r1, rs, nm), gg.y, be.y);
      r2 = fmaf(fmaf(r2, rs, nm), gg.z, be.z);
      r3 = fmaf(fmaf(r3, rs, nm), gg.w, be.w);
    }
    o0 += r0;
    o1 += r1;
    o2 += r2;
    o3 += r3;
  }
  uint2 out;
  out.x = pack_bf16x2(o0, o1);
  out.y = pack_bf16x2(o2, o3);
  return out;
}

template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int EPI, int ORDER>
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
  constexpr int CPR = BK / 8;       // 16-byte chunks per LDS row
  constexpr int RPC = 64 / CPR;     // rows one wave copy instruction fills
  constexpr int XI = BM / (RPC * NWAVES);  // copy instructions per wave per stage, X tile
  constexpr int WI = BN / (RPC * NWAVES);  // ... W tile
  constexpr int SSTAGE = (BM + BN) * CPR;  // 16-byte slots per stage buffer
  static_assert(XI * RPC * NWAVES == BM && WI * RPC * NWAVES == BN, "tile/wave mismatch");
  static_assert(BK == 32 || BK == 64, "16-byte chunk swizzles exist for 4 and 8 chunks per row");
  static_assert(CPR == 4 || NWAVES % 2 == 0, "copy slot phase needs an even wave count");
  static_assert(TN % 2 == 0 && STATS_WIDTH == 64, "epilogue passes are 64 features wide");
  // Buffer b holds X rows at smem[b*SSTAGE ..] and W rows after them.
  __shared__ u32x4 smem[2 * SSTAGE];
  // Per-feature vectors of the current tile (bias, then col_s or gamma and
  // beta), double-buffered by the parity of the workgroup's tile count.
  constexpr bool FOLD_ = EPI == EPI_FOLD || EPI == EPI_FOLD_GELU;
  constexpr bool LNRES_ = EPI == EPI_LNRES_STATS;
  constexpr int NV = 1 + (FOLD_ ? 1 : 0) + (LNRES_ ? 2 : 0);
  static_assert(NV <= NWAVES && BN <= 256, "one vector per wave copy");
  __shared__ float4 svec[2][NV][BN / 4];
  static_assert(XI >= 4, "a wave's epilogue region is 4 of its X copy slots");

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: kept in an SGPR
  const int l32 = lane & 31;
  const int lhi = lane >> 5;
  const int wn0 = (wave % WAVES_N) * WN;
  const int wm0 = (wave / WAVES_N) * WM;
  const int nkt = K / BK;
  const int G = gridDim.x;

  // Lane l of wave w, copy j, fills LDS slot p = (j*NWAVES + w)*64 + l of a
  // tile: row p / 8, stored chunk l % 8.  Its logical chunk
  // (l & 7) ^ (l >> 3) ^ (w & 1) is the same for every j; its rows are
  // NWAVES * 8 apart.
  constexpr int DSTEP = NWAVES * RPC;
  const int drow = wave * RPC + lane / CPR;
  const int dch = copy_chunk<CPR>(lane, wave);
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_address(smem) + wave * 64 * 16);
  constexpr uint32_t STAGE_BYTES = SSTAGE * 16;
  constexpr uint32_t COPY_BYTES = NWAVES * 64 * 16;

  // The copy stream runs two stages ahead of the MFMA work through this
  // workgroup's sequence of (tile, stage) pairs.  The issue cursor holds
  // the tile and stage to copy next and the source pointers of that tile;
  // advancing past a tile's last stage moves it to the workgroup's next
  // tile (that work stays off the path between a barrier and the MFMAs).
  int it_tile = blockIdx.x;  // < n_tiles: the grid is never larger than the tile count
  int it_kt = 0;
  // Copy sources: a wave-uniform tile base (scalar registers) plus a 32-bit
  // byte offset per lane that stays fixed while the tile's stages advance,
  // so a copy needs no per-lane address arithmetic (the launcher checks that
  // BM rows of K bf16 fit the 32-bit offset).
  const uint16_t* xs;  // X row block of the tile
  const uint16_t* ws;  // W feature block of the tile
  uint32_t xo[XI], wo[WI];
#pragma unroll
  for (int j = 0; j < WI; ++j) wo[j] = (uint32_t)((drow + j * DSTEP) * K + dch * 8) * 2u;
  auto point = [&]() {
    int tm_, tn_;
    tile_coords<ORDER>(it_tile, n_tiles, tiles_n, &tm_, &tn_);
    xs = X + (size_t)(tm_ * BM) * K;
    ws = W + (size_t)(tn_ * BN) * K;
#pragma unroll
    for (int j = 0; j < XI; ++j)  // rows past M: clamped, never stored
      xo[j] = (uint32_t)((min(tm_ * BM + drow + j * DSTEP, M - 1) - tm_ * BM) * K + dch * 8) * 2u;
  };
  auto issue = [&](int b) {
    if (it_tile >= n_tiles) return;
    const int ko = it_kt * BK;
    const uint32_t base = lds0 + (uint32_t)b * STAGE_BYTES;
    const uint16_t* sx = xs + ko;
    const uint16_t* sw = ws + ko;
#pragma unroll
    for (int j = 0; j < XI; ++j) copy_to_lds16_at(sx, xo[j], base + j * COPY_BYTES);
#pragma unroll
    for (int j = 0; j < WI; ++j) copy_to_lds16_at(sw, wo[j], base + BM * CPR * 16 + j * COPY_BYTES);
  };
  auto advance = [&]() {
    if (++it_kt == nkt) {
      it_kt = 0;
      it_tile += G;
      if (it_tile < n_tiles) point();
    }
  };

  int t = blockIdx.x;
  point();
  issue(0);
  advance();
  const bool second = it_tile < n_tiles;
  issue(1);
  advance();
  if (second)
    wait_copies<XI + WI>(1);
  else
    wait_copies<XI + WI>(0);
  __syncthreads();

  constexpr int S = BK / 16;   // 16-wide MFMA steps per stage
  constexpr int NR = TN + TM;  // fragment reads per step
  constexpr int NM = TN * TM;  // MFMAs per step
  static_assert(S % 2 == 0, "fragment parity must restart at every stage");
  static_assert(NM >= NR, "interleave needs at least one MFMA per read");
  bf16x8 fa[2][TN], fb[2][TM];
  int cur_buf = 0;
  int tpar = 0;

  for (;;) {
    int tm, tn;
    tile_coords<ORDER>(t, n_tiles, tiles_n, &tm, &tn);
    const int m0 = tm * BM;
    const int n0 = tn * BN;

    // This tile's per-feature vectors into svec[tpar], wave w copying
    // vector w (BN floats: one 16-byte chunk per lane).  The main loop's
    // first stage waits for every copy and meets at a barrier, so the
    // epilogue finds them in place; the buffer was last read by the
    // epilogue two tiles back.
    if (wave < NV && lane < BN / 4) {
      const float* src = bias;
      if constexpr (FOLD_) { if (wave == 1) src = ex.col_s; }
      if constexpr (LNRES_) { if (wave == 1) src = ex.gamma; if (wave == 2) src = ex.beta; }
      copy_lanes_to_lds16(src + n0, lds_address(&svec[tpar][wave][0]));
    }

    // LayerNorm factors of this lane's rows (fused LayerNorm epilogues),
    // fetched now so their latency hides behind the main loop.
    float2 rowf[TM];
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      rowf[j] = make_float2(0.0f, 0.0f);
      if constexpr (EPI == EPI_FOLD || EPI == EPI_FOLD_GELU || EPI == EPI_LNRES_STATS)
        rowf[j] = ex.rows_in[min(m0 + wm0 + j * 32 + l32, M - 1)];
    }

    f32x16 acc[TN][TM];
#pragma unroll
    for (int i = 0; i < TN; ++i)
#pragma unroll
      for (int j = 0; j < TM; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    {
      const u32x4* sx = smem + cur_buf * SSTAGE;
      const u32x4* sw = sx + BM * CPR;
#pragma unroll
      for (int i = 0; i < TN; ++i)
        fa[0][i] = __builtin_bit_cast(bf16x8, sw[swz<CPR>(wn0 + i * 32 + l32, lhi)]);
#pragma unroll
      for (int j = 0; j < TM; ++j)
        fb[0][j] = __builtin_bit_cast(bf16x8, sx[swz<CPR>(wm0 + j * 32 + l32, lhi)]);
    }

    // One stage per trip.  Steps 0 .. S-2 run their MFMAs with the fragment
    // reads of the following step interleaved one by one (pinned with
    // scheduling group barriers).  Then the wave waits for everything it
    // issued before (the copies of the next stage; at a tile's first stage
    // also the previous tile's epilogue loads and stores) and all waves
    // meet: the next stage is published and nobody reads this stage's
    // buffer any more, so the copies of the stage after next go into it.
    // The last step's MFMAs, which need no LDS, run after the barrier while
    // the first fragments of the next stage are read, so the MFMA pipe does
    // not wait for LDS at the stage boundary.  (At a tile's last stage those
    // reads are discarded; the next tile reads its own after the epilogue.)
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
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[cur][i], fb[cur][j], acc[i][j],
                                                                0, 0, 0);
      }
#pragma unroll
      for (int ks = 0; ks + 1 < S; ++ks) {
#pragma unroll
        for (int x = 0; x < NR; ++x) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NM - NR, 0);
      }
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // this stage's reads are done
      __syncthreads();
      const bool last_stage = kt == nkt - 1;
      if (!last_stage) issue(cur_buf);
      cur_buf ^= 1;
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
          acc[i][j] =
              __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[1][i], fb[1][j], acc[i][j], 0, 0, 0);
#pragma unroll
      for (int x = 0; x < NR; ++x) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, NM - NR, 0);
      if (!last_stage) advance();
    }

    // Epilogue, in passes over this wave's own 4 KB region (no other wave
    // touches it, so no barrier is needed).  Pass (j, ip) covers the 32
    // token rows of accumulator tile j and the 64 features of accumulator
    // tiles 2ip, 2ip+1, which is exactly one row-statistics partial.
    // acc[i][j] register r holds Y[m][n] with
    //   m = m0 + wm0 + j*32 + lane%32,
    //   n = n0 + wn0 + i*32 + 8*(r/4) + 4*(lane/32) + r%4,
    // i.e. registers 4g..4g+3 are unit 8*(i%2) + 2g + lane/32 of region row
    // lane%32.  Per pass:
    //   1. (residual modes) the pass's R rows, loaded for all passes with
    //      16-byte coalesced loads before the first, go into the region;
    //   2. each lane finishes its accumulators (reading its residual units
    //      back), rounds once to bf16 and writes the region; the statistics
    //      modes also sum the rounded values of its row;
    //   3. the region is stored as whole 128-byte row segments.
    {
      constexpr bool FOLD = EPI == EPI_FOLD || EPI == EPI_FOLD_GELU;
      constexpr bool RES =
          EPI == EPI_BIAS_RESIDUAL || EPI == EPI_RES_STATS || EPI == EPI_LNRES_STATS;
      constexpr bool LNRES = EPI == EPI_LNRES_STATS;
      constexpr bool STATS = EPI == EPI_RES_STATS || EPI == EPI_LNRES_STATS;
      constexpr int PW = STATS_WIDTH;
      constexpr int NP = TM * (TN / 2);  // passes
      // Region row r lives in this wave's X copy slot r/8 of the buffer the
      // last stage released (8 rows of 128 bytes per 1 KB slot).
      u32x4* const rbase = smem + (cur_buf ^ 1) * SSTAGE + wave * 64;
      auto slot16 = [&](int r, int s16) -> u32x4* {
        return rbase + (r >> 3) * (NWAVES * 64) + (r & 7) * 8 + s16;
      };
      auto cell8 = [&](int r, int u) -> uint2* {
        return reinterpret_cast<uint2*>(slot16(r, 0)) + u;
      };
      const int cr = lane >> 3;  // row within the 8 rows of one coalesced access
      const int cp = lane & 7;   // 16-byte pair within a row

      u32x4 rv[RES ? NP : 1][4];
      if constexpr (RES) {
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          const int j = p / (TN / 2), ip = p % (TN / 2);
#pragma unroll
          for (int it = 0; it < 4; ++it) {
            const int m = min(m0 + wm0 + j * 32 + it * 8 + cr, M - 1);
            rv[p][it] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(
                R + (size_t)m * N + n0 + wn0 + ip * 64 + 8 * cp));
          }
        }
      }
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        const int j = p / (TN / 2), ip = p % (TN / 2);
        const float rs = rowf[j].x, nm = rowf[j].y;
        if constexpr (RES) {
#pragma unroll
          for (int it = 0; it < 4; ++it) {
            const int r = it * 8 + cr;
            const int ph = (2 * cp) ^ rsw(r);  // physical unit of logical unit 2cp
            u32x4 v = rv[p][it];
            if (ph & 1) v = u32x4{v[2], v[3], v[0], v[1]};
            *slot16(r, ph >> 1) = v;
          }
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        }
        float st_s = 0.0f, st_q = 0.0f;
#pragma unroll
        for (int ii = 0; ii < 2; ++ii) {
          const int i = 2 * ip + ii;
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int f = n0 + wn0 + i * 32 + 8 * g + 4 * lhi;  // first of the 4 features
            const int fq = (f - n0) >> 2;  // float4 index within the tile
            const float4 bb = svec[tpar][0][fq];
            float4 cs = {0.0f, 0.0f, 0.0f, 0.0f}, gg = cs, be = cs;
            if constexpr (FOLD) cs = svec[tpar][1][fq];
            if constexpr (LNRES) {
              gg = svec[tpar][1][fq];
              be = svec[tpar][2][fq];
            }
            uint2& cell = *cell8(l32, (8 * ii + 2 * g + lhi) ^ rsw(l32));
            const float a[4] = {acc[i][j][4 * g + 0], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                                acc[i][j][4 * g + 3]};
            const uint2 out = finish4<EPI>(a, bb, cs, gg, be, rs, nm, RES ? cell : uint2{0u, 0u});
            cell = out;
            if constexpr (STATS) {
              const float v0 = __uint_as_float(out.x << 16), v1 = __uint_as_float(out.x & 0xffff0000u);
              const float v2 = __uint_as_float(out.y << 16), v3 = __uint_as_float(out.y & 0xffff0000u);
              st_s += (v0 + v1) + (v2 + v3);
              st_q = fmaf(v0, v0, fmaf(v1, v1, fmaf(v2, v2, fmaf(v3, v3, st_q))));
            }
          }
        }
        if constexpr (STATS) {
          // The lane and its partner (lane ^ 32) hold complementary halves
          // of the row's 64 features; partial index = first feature / 64.
          const float s1 = st_s + __shfl_xor(st_s, 32, 64);
          const float q1 = st_q + __shfl_xor(st_q, 32, 64);
          const int m = m0 + wm0 + j * 32 + l32;
          if (lhi == 0 && m < M) {
            constexpr float inv_w = 1.0f / (float)PW;
            const float mean = s1 * inv_w;
            ex.stats_out[(size_t)((n0 + wn0) / PW + ip) * M + m] =
                make_float2(mean, fmaxf(q1 * inv_w - mean * mean, 0.0f));
          }
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // region written by all lanes
        u32x4 ov[4];
#pragma unroll
        for (int it = 0; it < 4; ++it) {
          const int r = it * 8 + cr;
          const int ph = (2 * cp) ^ rsw(r);
          ov[it] = *slot16(r, ph >> 1);
          if (ph & 1) ov[it] = u32x4{ov[it][2], ov[it][3], ov[it][0], ov[it][1]};
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // region free for the next pass
#pragma unroll
        for (int it = 0; it < 4; ++it) {
          const int m = m0 + wm0 + j * 32 + it * 8 + cr;
          if (m < M)
            __builtin_nontemporal_store(
                ov[it], reinterpret_cast<u32x4*>(Y + (size_t)m * N + n0 + wn0 + ip * 64 + 8 * cp));
        }
      }
    }

    // The region's reads are done (waited above); this wave's deferred copies
    // of the next tile's second stage go into the same slots.
    issue(cur_buf ^ 1);
    advance();
    tpar ^= 1;
    t += G;
    if (t >= n_tiles) break;
  }
}

template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int PER_CU>
hipError_t launch_tiles(const uint16_t* X, const uint16_t* W, const float* bias, const uint16_t* R,
                        uint16_t* Y, int64_t M, int N, int K, int epi, const LinearExtra& ex,
                        hipStream_t stream) {
  if ((int64_t)BM * K * 2 > (int64_t)UINT32_MAX) return hipErrorInvalidValue;  // copy offsets
  int cus = ex.n_cus;
  if (cus <= 0) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
  }
  const int tiles_n = N / BN;
  const int64_t tiles_m = (M + BM - 1) / BM;
  const int n_tiles = (int)(tiles_m * tiles_n);
  const dim3 grid((unsigned)std::min<int64_t>(n_tiles, (int64_t)cus * PER_CU));
  const dim3 block(WAVES_M * WAVES_N * 64);
#define SURGE_LAUNCH_EPI(E, O)                                                                   \
  hipLaunchKernelGGL((linear_bf16_kernel<BM, BN, BK, WAVES_M, WAVES_N, E, O>), grid, block, 0, stream, \
                     X, W, bias, R, Y, (int)M, N, K, tiles_n, n_tiles, ex)
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
// 64 tokens x 128 features, one workgroup per CU) where the feature count
// allows it and there are enough token rows to fill the chip; 128 x 128
// tiles (4 waves of 64 x 64, two workgroups per CU) otherwise.
static bool big_tiles(int64_t M, int N) { return N % 256 == 0 && M >= 8192; }

int linear_stats_width(int64_t, int) { return STATS_WIDTH; }

hipError_t launch_linear(const uint16_t* X, const uint16_t* W, const float* bias, const uint16_t* R,
                         uint16_t* Y, int64_t M, int N, int K, int epi, const LinearExtra& ex,
                         hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  if (big_tiles(M, N))
    return launch_tiles<256, 256, 64, 4, 2, 1>(X, W, bias, R, Y, M, N, K, epi, ex, stream);
  return launch_tiles<128, 128, 64, 2, 2, 2>(X, W, bias, R, Y, M, N, K, epi, ex, stream);
}

}  // namespace surge
