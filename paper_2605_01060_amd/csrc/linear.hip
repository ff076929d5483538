// Token-major linear layers on bf16 MFMA (gfx950): Y = epi(X W^T + b).
//
// X is the packed token matrix [M, K] (M = tokens of the chunk, no padding),
// W the layer weight repacked to [N, K] so both operands are K-contiguous.
//
// Tiling.  A workgroup computes a BM x BN tile of Y (tokens x features) with
// WAVES_M x WAVES_N waves; each wave owns a (BM/WAVES_M) x (BN/WAVES_N)
// sub-tile held as 32 x 32 v_mfma_f32_32x32x16_bf16 accumulators.  K is
// walked in 64-wide stages through a double-buffered LDS tile.
//
// Staging.  Each thread loads its share of stage k+1 (16-byte chunks) into
// registers while stage k runs on the MFMA units, then writes it to the
// other LDS buffer; one barrier per stage.  LDS rows are 128 B (64 bf16 of
// K); the 16-byte chunk c of row r is stored at position
// c ^ (r & 7) ^ ((r >> 3) & 1).  A fragment read takes the same chunk from
// consecutive rows: any 8 aligned rows then land on 8 different 16-byte
// positions and any 16 aligned rows on 16 different (row parity, position)
// pairs, so the reads are free of bank conflicts whether the LDS serves a
// 16-byte read 8 lanes at a time over 32 banks or 16 lanes at a time over
// 64 banks.  Row writes (8 lanes per row, all chunks) are contiguous.
//
// Operand roles.  The MFMA A operand is the weight tile and B the token
// tile, so the accumulators hold Y^T: each lane owns one token row and four
// consecutive features per register group, which makes the epilogue (bias,
// GELU, residual, bf16 store) 8-byte vector accesses.
//
// Order.  Workgroups are dispatched round-robin over the 8 XCDs; the tile
// index is remapped so each XCD walks a contiguous range of token-row
// blocks, all feature tiles of a row block back to back, keeping that row
// block in the XCD's L2 while its feature tiles run.
//
// Every output row is computed from its own input row with a fixed K order
// (no split-K, no atomics), so a text's result does not depend on which
// other texts share its SuperBatch or chunk.
#include "device_common.h"
#include "kernels.h"

namespace surge {
namespace {

constexpr int BK = 64;

__device__ __forceinline__ int swz(int row, int chunk) {
  return row * 8 + (chunk ^ (row & 7) ^ ((row >> 3) & 1));
}

// Direct global -> LDS copy of 16 bytes per lane (gfx950 global_load_lds):
// the wave's 64 lanes land contiguously at LDS byte address `lds` (wave
// uniform, passed in M0).  Issued as inline assembly so that the waits are
// placed by the kernel itself (s_waitcnt vmcnt before the barrier that
// publishes a stage); the compiler cannot prove which stage an in-flight
// copy targets and would otherwise wait for it before every LDS read.
__device__ __forceinline__ void copy_to_lds16(const void* g, uint32_t lds) {
  asm volatile(
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, off"
      :
      : "v"(g), "s"(lds)
      : "memory", "m0");
}

__device__ __forceinline__ void wait_copies() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

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

__device__ __forceinline__ uint32_t lds_address(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

template <int BM, int BN, int WAVES_M, int WAVES_N, int EPI, bool DTL, int ORDER>
__global__ __launch_bounds__(WAVES_M* WAVES_N * 64) void linear_bf16_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W, const float* __restrict__ bias,
    const uint16_t* __restrict__ R, uint16_t* __restrict__ Y, int M, int N, int K, int tiles_n,
    int n_tiles) {
  constexpr int NWAVES = WAVES_M * WAVES_N;
  constexpr int WM = BM / WAVES_M;  // tokens per wave
  constexpr int WN = BN / WAVES_N;  // features per wave
  constexpr int TM = WM / 32;       // 32-token accumulator tiles per wave
  constexpr int TN = WN / 32;       // 32-feature accumulator tiles per wave
  constexpr int NT = NWAVES * 64;
  constexpr int XI = BM * 8 / NT;  // 16-byte chunks per thread per stage, X tile
  constexpr int WI = BN * 8 / NT;  // ... W tile
  static_assert(XI * NT == BM * 8 && WI * NT == BN * 8, "tile/thread mismatch");
  static_assert(NT % 128 == 0, "a thread's rows must share their phase mod 16");

  // Main loop: stage b holds X rows at smem[b*SSTAGE ..] and W rows after
  // them.  Epilogue: the same memory holds fp32 output rows.
  constexpr int SSTAGE = (BM + BN) * 8;
  __shared__ u32x4 smem[2 * SSTAGE];
#define SX(b) (smem + (b) * SSTAGE)
#define SW(b) (smem + (b) * SSTAGE + BM * 8)

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;

  int tn, tm;
  tile_coords<ORDER>(blockIdx.x, n_tiles, tiles_n, &tm, &tn);
  const int m0 = tm * BM;
  const int n0 = tn * BN;
  const int wn0 = (wave % WAVES_N) * WN;
  const int wm0 = (wave / WAVES_N) * WM;

  // Thread t copies chunks t, t + NT, ... of each tile: chunk c is row c/8,
  // logical 16-byte column c%8.  NT is a multiple of 128, so every chunk of
  // a thread has the same column and the same row phase (row & 15), and its
  // rows are NT/8 apart: its LDS slots are s_idx0 + j * NT.
  constexpr int RSTEP = NT / 8;
  const int row0 = threadIdx.x >> 3;
  const int kc = threadIdx.x & 7;
  const int s_idx0 = swz(row0, kc);
  const u32x4* gw0 = reinterpret_cast<const u32x4*>(W + (size_t)(n0 + row0) * K) + kc;
  const size_t wstep = (size_t)RSTEP * K / 8;  // 16-byte units between a thread's W rows
  size_t xoff[XI];
#pragma unroll
  for (int j = 0; j < XI; ++j) {
    const int xrow = min(m0 + row0 + j * RSTEP, M - 1);  // rows past M read clamped, never stored
    xoff[j] = (size_t)xrow * (K / 8) + kc;
  }
  const u32x4* X4 = reinterpret_cast<const u32x4*>(X);

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

  if constexpr (DTL) {
    // Lane l of wave w, copy j, fills LDS slot p = (j*NWAVES + w)*64 + l of
    // a tile: row p/8, stored chunk l%8.  Its logical chunk is
    // (l%8) ^ (row&7) ^ ((row>>3)&1) = (l%8) ^ (l/8) ^ (w&1), the same for
    // every j (NWAVES is even); its rows are NWAVES*8 apart.
    constexpr int DSTEP = NWAVES * 8;
    const int drow = wave * 8 + (lane >> 3);
    const int dch = (lane & 7) ^ (lane >> 3) ^ (wave & 1);
    const uint16_t* xg[XI];
#pragma unroll
    for (int j = 0; j < XI; ++j)
      xg[j] = X + (size_t)min(m0 + drow + j * DSTEP, M - 1) * K + dch * 8;
    const uint16_t* wg = W + (size_t)(n0 + drow) * K + dch * 8;
    const size_t wgstep = (size_t)DSTEP * K;
    const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_address(smem) + wave * 64 * 16);
    constexpr uint32_t STAGE_BYTES = SSTAGE * 16;
    constexpr uint32_t COPY_BYTES = NWAVES * 64 * 16;

#define SURGE_ISSUE_STAGE(kk_, b_)                                                              \
    do {                                                                                        \
      const int ko_ = (kk_) * BK;                                                               \
      const uint32_t base_ = lds0 + (uint32_t)(b_) * STAGE_BYTES;                               \
      _Pragma("unroll") for (int j = 0; j < XI; ++j)                                            \
        copy_to_lds16(xg[j] + ko_, base_ + j * COPY_BYTES);                                     \
      _Pragma("unroll") for (int j = 0; j < WI; ++j)                                            \
        copy_to_lds16(wg + j * wgstep + ko_, base_ + BM * 8 * 16 + j * COPY_BYTES);             \
    } while (0)

    SURGE_ISSUE_STAGE(0, 0);
    wait_copies();
    __syncthreads();
    constexpr int NR = TN + TM;
    constexpr int NM = TN * TM;
    static_assert(NM >= NR, "interleave needs at least one MFMA per read");
    for (int kt = 0; kt < nkt; ++kt) {
      const int buf = kt & 1;
      if (kt + 1 < nkt) SURGE_ISSUE_STAGE(kt + 1, buf ^ 1);
      bf16x8 fa[2][TN], fb[2][TM];
#pragma unroll
      for (int i = 0; i < TN; ++i)
        fa[0][i] = __builtin_bit_cast(bf16x8, SW(buf)[swz(wn0 + i * 32 + l32, lhi)]);
#pragma unroll
      for (int j = 0; j < TM; ++j)
        fb[0][j] = __builtin_bit_cast(bf16x8, SX(buf)[swz(wm0 + j * 32 + l32, lhi)]);
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        const int cur = ks & 1;
        if (ks + 1 < BK / 16) {
          const int ch = (ks + 1) * 2 + lhi;
#pragma unroll
          for (int i = 0; i < TN; ++i)
            fa[cur ^ 1][i] = __builtin_bit_cast(bf16x8, SW(buf)[swz(wn0 + i * 32 + l32, ch)]);
#pragma unroll
          for (int j = 0; j < TM; ++j)
            fb[cur ^ 1][j] = __builtin_bit_cast(bf16x8, SX(buf)[swz(wm0 + j * 32 + l32, ch)]);
        }
#pragma unroll
        for (int i = 0; i < TN; ++i)
#pragma unroll
          for (int j = 0; j < TM; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[cur][i], fb[cur][j], acc[i][j],
                                                                0, 0, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);
#pragma unroll
      for (int ks = 0; ks + 1 < BK / 16; ++ks) {
#pragma unroll
        for (int t = 0; t < NR; ++t) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NM - NR, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
      wait_copies();
      __syncthreads();
    }
#undef SURGE_ISSUE_STAGE
  } else {
  u32x4 rx[XI], rw[WI];
#pragma unroll
  for (int j = 0; j < XI; ++j) rx[j] = X4[xoff[j]];
#pragma unroll
  for (int j = 0; j < WI; ++j) rw[j] = gw0[j * wstep];
#pragma unroll
  for (int j = 0; j < XI; ++j) SX(0)[s_idx0 + j * NT] = rx[j];
#pragma unroll
  for (int j = 0; j < WI; ++j) SW(0)[s_idx0 + j * NT] = rw[j];
  __syncthreads();

  // One 64-wide K stage per trip.  The body is branch-free (the last trip
  // re-loads its own stage into the idle buffer) so that the instruction
  // order below, pinned with scheduling group barriers, holds:
  //   global loads of stage k+1 | LDS reads of step 0 |
  //   steps 0..2: each MFMA followed by one LDS read of the next step |
  //   step 3 MFMAs | LDS writes of stage k+1.
  constexpr int NR = TN + TM;   // fragment reads per 16-wide step
  constexpr int NM = TN * TM;   // MFMAs per step
  static_assert(NM >= NR, "interleave needs at least one MFMA per read");
  for (int kt = 0; kt < nkt; ++kt) {
    const int buf = kt & 1;
    const int k8 = min(kt + 1, nkt - 1) * (BK / 8);
#pragma unroll
    for (int j = 0; j < XI; ++j) rx[j] = X4[xoff[j] + k8];
#pragma unroll
    for (int j = 0; j < WI; ++j) rw[j] = gw0[j * wstep + k8];

    bf16x8 fa[2][TN], fb[2][TM];
#pragma unroll
    for (int i = 0; i < TN; ++i)
      fa[0][i] = __builtin_bit_cast(bf16x8, SW(buf)[swz(wn0 + i * 32 + l32, lhi)]);
#pragma unroll
    for (int j = 0; j < TM; ++j)
      fb[0][j] = __builtin_bit_cast(bf16x8, SX(buf)[swz(wm0 + j * 32 + l32, lhi)]);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int cur = ks & 1;
      if (ks + 1 < BK / 16) {
        const int ch = (ks + 1) * 2 + lhi;
#pragma unroll
        for (int i = 0; i < TN; ++i)
          fa[cur ^ 1][i] = __builtin_bit_cast(bf16x8, SW(buf)[swz(wn0 + i * 32 + l32, ch)]);
#pragma unroll
        for (int j = 0; j < TM; ++j)
          fb[cur ^ 1][j] = __builtin_bit_cast(bf16x8, SX(buf)[swz(wm0 + j * 32 + l32, ch)]);
      }
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j)
          acc[i][j] =
              __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[cur][i], fb[cur][j], acc[i][j], 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < XI; ++j) SX(buf ^ 1)[s_idx0 + j * NT] = rx[j];
#pragma unroll
    for (int j = 0; j < WI; ++j) SW(buf ^ 1)[s_idx0 + j * NT] = rw[j];

    // Pin the order described above.
    __builtin_amdgcn_sched_group_barrier(0x020, XI + WI, 0);  // global loads
    __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);       // LDS reads, step 0
#pragma unroll
    for (int ks = 0; ks + 1 < BK / 16; ++ks) {
#pragma unroll
      for (int t = 0; t < NR; ++t) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
      }
      __builtin_amdgcn_sched_group_barrier(0x008, NM - NR, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);       // last step
    __builtin_amdgcn_sched_group_barrier(0x200, XI + WI, 0);  // LDS writes
    __syncthreads();
  }

  }

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
  //   1. (residual only) every thread copies whole rows of R into the tile
  //      with 16-byte coalesced loads, all issued before any is used;
  //   2. each lane adds bias (+ GELU) to its accumulators, adds the residual
  //      read back from the tile, rounds once to bf16 and writes the tile;
  //   3. every thread stores whole rows of the tile with 16-byte stores.
#undef SX
#undef SW
  {
    static_assert(2 * (BM + BN) * 8 * 16 >= BM * BN * 2, "bf16 tile must fit the LDS");
    constexpr int U = BN / 4;            // 8-byte units per row
    constexpr int PAIRS = BN / 8;        // 16-byte pairs per row
    constexpr int RPI = NT / PAIRS;      // rows per coalesced iteration
    constexpr int ITER = BM / RPI;
    static_assert(BM % RPI == 0 && U >= 32, "epilogue shape");
    uint2* t8 = reinterpret_cast<uint2*>(smem);
    u32x4* t16 = smem;
    const int cp = threadIdx.x % PAIRS;  // this thread's 16-byte pair in a row
    const int cr = threadIdx.x / PAIRS;
    if (EPI == EPI_BIAS_RESIDUAL) {
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
#pragma unroll
    for (int i = 0; i < TN; ++i) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int u = (wn0 + i * 32 + 8 * g) / 4 + lhi;
        const float4 bb = *reinterpret_cast<const float4*>(bias + n0 + 4 * u);
#pragma unroll
        for (int j = 0; j < TM; ++j) {
          const int r = wm0 + j * 32 + l32;
          float o0 = acc[i][j][4 * g + 0] + bb.x;
          float o1 = acc[i][j][4 * g + 1] + bb.y;
          float o2 = acc[i][j][4 * g + 2] + bb.z;
          float o3 = acc[i][j][4 * g + 3] + bb.w;
          if (EPI == EPI_BIAS_GELU) {
            o0 = gelu_erf(o0);
            o1 = gelu_erf(o1);
            o2 = gelu_erf(o2);
            o3 = gelu_erf(o3);
          }
          uint2& cell = t8[r * U + (u ^ (r & 31))];
          if (EPI == EPI_BIAS_RESIDUAL) {
            const uint2 rr = cell;
            o0 += __uint_as_float(rr.x << 16);
            o1 += __uint_as_float(rr.x & 0xffff0000u);
            o2 += __uint_as_float(rr.y << 16);
            o3 += __uint_as_float(rr.y & 0xffff0000u);
          }
          uint2 out;
          out.x = pack_bf16x2(o0, o1);
          out.y = pack_bf16x2(o2, o3);
          cell = out;
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

template <int BM, int BN, int WAVES_M, int WAVES_N, bool DTL>
hipError_t launch_tiles(const uint16_t* X, const uint16_t* W, const float* bias, const uint16_t* R,
                        uint16_t* Y, int64_t M, int N, int K, int epi, hipStream_t stream) {
  const int tiles_n = N / BN;
  const int64_t tiles_m = (M + BM - 1) / BM;
  const int n_tiles = (int)(tiles_m * tiles_n);
  const dim3 grid((unsigned)n_tiles);
  const dim3 block(WAVES_M * WAVES_N * 64);
  switch (epi) {
    case EPI_BIAS:
      hipLaunchKernelGGL((linear_bf16_kernel<BM, BN, WAVES_M, WAVES_N, EPI_BIAS, DTL, ORDER_ROW_GROUPS>),
                         grid, block, 0, stream, X, W, bias, R, Y, (int)M, N, K, tiles_n, n_tiles);
      break;
    case EPI_BIAS_GELU:
      hipLaunchKernelGGL(
          (linear_bf16_kernel<BM, BN, WAVES_M, WAVES_N, EPI_BIAS_GELU, DTL, ORDER_FEATURE_HALVES>), grid,
          block, 0, stream, X, W, bias, R, Y, (int)M, N, K, tiles_n, n_tiles);
      break;
    default:
      hipLaunchKernelGGL(
          (linear_bf16_kernel<BM, BN, WAVES_M, WAVES_N, EPI_BIAS_RESIDUAL, DTL, ORDER_ROW_GROUPS>), grid,
          block, 0, stream, X, W, bias, R, Y, (int)M, N, K, tiles_n, n_tiles);
      break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_linear(const uint16_t* X, const uint16_t* W, const float* bias, const uint16_t* R,
                         uint16_t* Y, int64_t M, int N, int K, int epi, hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  // 256 x 256 tiles (8 waves of 64 tokens x 128 features) where the feature
  // count allows it and there are enough token rows to fill the chip;
  // 128 x 128 tiles (4 waves of 64 x 64) otherwise.
  if (N % 256 == 0 && M >= 8192)
    return launch_tiles<256, 256, 4, 2, true>(X, W, bias, R, Y, M, N, K, epi, stream);
  return launch_tiles<128, 128, 2, 2, true>(X, W, bias, R, Y, M, N, K, epi, stream);
}

}  // namespace surge
