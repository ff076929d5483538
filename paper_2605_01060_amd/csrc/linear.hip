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
// K); the 16-byte chunk c of row r is stored at position c ^ (r & 7), so the
// fragment reads (8 consecutive rows, same chunk) and the row writes hit
// distinct banks.
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

// Native 16-byte vector (HIP's uint4 is a union-based struct, which keeps
// LLVM from turning the staging arrays into registers).
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

template <int BM, int BN, int WAVES_M, int WAVES_N, int EPI>
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

  __shared__ u32x4 sX[2][BM * 8];
  __shared__ u32x4 sW[2][BN * 8];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;

  // XCD-aware tile order (see header).
  int tile = blockIdx.x;
  {
    const int per_xcd = n_tiles >> 3;
    const int full = per_xcd << 3;
    if (tile < full) tile = (tile & 7) * per_xcd + (tile >> 3);
  }
  const int tn = tile % tiles_n;
  const int tm = tile / tiles_n;
  const int m0 = tm * BM;
  const int n0 = tn * BN;
  const int wn0 = (wave % WAVES_N) * WN;
  const int wm0 = (wave / WAVES_N) * WM;

  // Thread t copies chunks t, t + NT, ... of each tile: chunk c is row c/8,
  // logical 16-byte column c%8, stored at column (c%8) ^ (row & 7).  NT is a
  // multiple of 64, so every chunk of a thread has the same column and the
  // same row phase, and its rows are NT/8 apart.
  constexpr int RSTEP = NT / 8;
  const int row0 = threadIdx.x >> 3;
  const int kc = threadIdx.x & 7;
  const int s_idx0 = row0 * 8 + (kc ^ (row0 & 7));
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

  u32x4 rx[XI], rw[WI];
#pragma unroll
  for (int j = 0; j < XI; ++j) rx[j] = X4[xoff[j]];
#pragma unroll
  for (int j = 0; j < WI; ++j) rw[j] = gw0[j * wstep];
#pragma unroll
  for (int j = 0; j < XI; ++j) sX[0][s_idx0 + j * NT] = rx[j];
#pragma unroll
  for (int j = 0; j < WI; ++j) sW[0][s_idx0 + j * NT] = rw[j];
  __syncthreads();

  for (int kt = 0; kt < nkt; ++kt) {
    const int buf = kt & 1;
    const bool more = kt + 1 < nkt;
    if (more) {
      const int k8 = (kt + 1) * (BK / 8);
#pragma unroll
      for (int j = 0; j < XI; ++j) rx[j] = X4[xoff[j] + k8];
#pragma unroll
      for (int j = 0; j < WI; ++j) rw[j] = gw0[j * wstep + k8];
    }
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int ch = ks * 2 + lhi;
      bf16x8 a[TN], b[TM];
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int row = wn0 + i * 32 + l32;
        a[i] = __builtin_bit_cast(bf16x8, sW[buf][row * 8 + (ch ^ (row & 7))]);
      }
#pragma unroll
      for (int j = 0; j < TM; ++j) {
        const int row = wm0 + j * 32 + l32;
        b[j] = __builtin_bit_cast(bf16x8, sX[buf][row * 8 + (ch ^ (row & 7))]);
      }
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
#pragma unroll
      for (int j = 0; j < XI; ++j) sX[buf ^ 1][s_idx0 + j * NT] = rx[j];
#pragma unroll
      for (int j = 0; j < WI; ++j) sW[buf ^ 1][s_idx0 + j * NT] = rw[j];
    }
    __syncthreads();
  }

  // Epilogue.  acc[i][j] register r holds Y[m][n] with
  //   m = m0 + wm0 + j*32 + lane%32
  //   n = n0 + wn0 + i*32 + 8*(r/4) + 4*(lane/32) + r%4.
#pragma unroll
  for (int j = 0; j < TM; ++j) {
    const int m = m0 + wm0 + j * 32 + l32;
    if (m >= M) continue;
#pragma unroll
    for (int i = 0; i < TN; ++i) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = n0 + wn0 + i * 32 + g * 8 + lhi * 4;
        const float4 bb = *reinterpret_cast<const float4*>(bias + n);
        float v0 = acc[i][j][g * 4 + 0] + bb.x;
        float v1 = acc[i][j][g * 4 + 1] + bb.y;
        float v2 = acc[i][j][g * 4 + 2] + bb.z;
        float v3 = acc[i][j][g * 4 + 3] + bb.w;
        if (EPI == EPI_BIAS_GELU) {
          v0 = gelu_erf(v0);
          v1 = gelu_erf(v1);
          v2 = gelu_erf(v2);
          v3 = gelu_erf(v3);
        }
        const size_t o = (size_t)m * N + n;
        if (EPI == EPI_BIAS_RESIDUAL) {
          const uint2 rr = *reinterpret_cast<const uint2*>(R + o);
          v0 += __uint_as_float(rr.x << 16);
          v1 += __uint_as_float(rr.x & 0xffff0000u);
          v2 += __uint_as_float(rr.y << 16);
          v3 += __uint_as_float(rr.y & 0xffff0000u);
        }
        uint2 out;
        out.x = pack_bf16x2(v0, v1);
        out.y = pack_bf16x2(v2, v3);
        *reinterpret_cast<uint2*>(Y + o) = out;
      }
    }
  }
}

template <int BM, int BN, int WAVES_M, int WAVES_N>
hipError_t launch_tiles(const uint16_t* X, const uint16_t* W, const float* bias, const uint16_t* R,
                        uint16_t* Y, int64_t M, int N, int K, int epi, hipStream_t stream) {
  const int tiles_n = N / BN;
  const int64_t tiles_m = (M + BM - 1) / BM;
  const int n_tiles = (int)(tiles_m * tiles_n);
  const dim3 grid((unsigned)n_tiles);
  const dim3 block(WAVES_M * WAVES_N * 64);
  switch (epi) {
    case EPI_BIAS:
      hipLaunchKernelGGL((linear_bf16_kernel<BM, BN, WAVES_M, WAVES_N, EPI_BIAS>), grid, block, 0,
                         stream, X, W, bias, R, Y, (int)M, N, K, tiles_n, n_tiles);
      break;
    case EPI_BIAS_GELU:
      hipLaunchKernelGGL((linear_bf16_kernel<BM, BN, WAVES_M, WAVES_N, EPI_BIAS_GELU>), grid,
                         block, 0, stream, X, W, bias, R, Y, (int)M, N, K, tiles_n, n_tiles);
      break;
    default:
      hipLaunchKernelGGL((linear_bf16_kernel<BM, BN, WAVES_M, WAVES_N, EPI_BIAS_RESIDUAL>), grid,
                         block, 0, stream, X, W, bias, R, Y, (int)M, N, K, tiles_n, n_tiles);
      break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_linear(const uint16_t* X, const uint16_t* W, const float* bias, const uint16_t* R,
                         uint16_t* Y, int64_t M, int N, int K, int epi, hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  // 256 x 256 tiles (8 waves of 128 tokens x 64 features) where the feature
  // count allows it and there are enough token rows to fill the chip;
  // 128 x 128 tiles (4 waves of 64 x 64) otherwise.
  if (N % 256 == 0 && M >= 8192)
    return launch_tiles<256, 256, 2, 4>(X, W, bias, R, Y, M, N, K, epi, stream);
  return launch_tiles<128, 128, 2, 2>(X, W, bias, R, Y, M, N, K, epi, stream);
}

}  // namespace surge
