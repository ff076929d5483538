// Token-major linear layers on bf16 MFMA (gfx950): Y = epi(X W^T + b).
//
// X is the packed token matrix [M, K] (M = tokens of the chunk, no padding),
// W the layer weight repacked to [N, K] so both operands are K-contiguous.
// One workgroup (4 waves) computes a 128 x 128 tile of Y; each wave owns a
// 64 x 64 sub-tile as 2 x 2 v_mfma_f32_32x32x16_bf16 accumulators.  K is
// walked in 64-wide steps staged through LDS with a double buffer: the
// global loads of step k+1 are in flight while step k runs on the MFMA
// units.  LDS rows are 128 bytes; the 16-byte chunk index is XOR-swizzled
// with the row so that the 16-byte fragment reads of 8 consecutive rows hit
// distinct banks.
//
// The MFMA's A operand is the weight tile and its B operand the token tile,
// so the accumulator holds Y^T: each lane owns one token row and four
// consecutive output features per register group, which makes the epilogue
// (bias, GELU, residual, bf16 store) 8-byte vector loads and stores.
//
// Every output row is computed from its own input row with a fixed K order
// (no split-K, no atomics), so a text's result does not depend on which
// other texts share its SuperBatch.
#include "device_common.h"
#include "kernels.h"

namespace surge {
namespace {

constexpr int BM = 128;  // tokens per tile
constexpr int BN = 128;  // output features per tile
constexpr int BK = 64;   // K per LDS stage
constexpr int THREADS = 256;
constexpr int CHUNKS = BM * BK / 8 / THREADS;  // 16-byte chunks per thread per operand (= 4)

template <int EPI>
__global__ __launch_bounds__(THREADS, 2) void linear_bf16_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W, const float* __restrict__ bias,
    const uint16_t* __restrict__ R, uint16_t* __restrict__ Y, int M, int N, int K, int tiles_n) {
  __shared__ uint4 sX[2][BM * BK / 8];
  __shared__ uint4 sW[2][BN * BK / 8];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int tn = blockIdx.x % tiles_n;
  const int tm = blockIdx.x / tiles_n;
  const int m0 = tm * BM;
  const int n0 = tn * BN;
  const int wn = (wave & 1) * 64;   // wave's feature offset in the tile
  const int wm = (wave >> 1) * 64;  // wave's token offset in the tile

  // Global -> LDS mapping: chunk c of a tile is row c / 8, 16-byte column c % 8.
  const uint4* gX[CHUNKS];
  const uint4* gW[CHUNKS];
  int sidx[CHUNKS];
#pragma unroll
  for (int c = 0; c < CHUNKS; ++c) {
    const int idx = tid + c * THREADS;
    const int row = idx >> 3;
    const int kc = idx & 7;
    const int xrow = min(m0 + row, M - 1);  // rows past M are read clamped, never stored
    gX[c] = reinterpret_cast<const uint4*>(X + (size_t)xrow * K) + kc;
    gW[c] = reinterpret_cast<const uint4*>(W + (size_t)(n0 + row) * K) + kc;
    sidx[c] = row * 8 + (kc ^ (row & 7));
  }

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  uint4 rx[CHUNKS], rw[CHUNKS];
#pragma unroll
  for (int c = 0; c < CHUNKS; ++c) {
    rx[c] = gX[c][0];
    rw[c] = gW[c][0];
  }
#pragma unroll
  for (int c = 0; c < CHUNKS; ++c) {
    sX[0][sidx[c]] = rx[c];
    sW[0][sidx[c]] = rw[c];
  }
  __syncthreads();

  const int nkt = K / BK;
  const int l32 = lane & 31;
  const int lhi = lane >> 5;
  for (int kt = 0; kt < nkt; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nkt) {
      const int off = (kt + 1) * (BK / 8);
#pragma unroll
      for (int c = 0; c < CHUNKS; ++c) {
        rx[c] = gX[c][off];
        rw[c] = gW[c][off];
      }
    }
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int ch = ks * 2 + lhi;
      bf16x8 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int row = wn + i * 32 + l32;
        a[i] = as_bf16x8(sW[buf][row * 8 + (ch ^ (row & 7))]);
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int row = wm + j * 32 + l32;
        b[j] = as_bf16x8(sX[buf][row * 8 + (ch ^ (row & 7))]);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nkt) {
#pragma unroll
      for (int c = 0; c < CHUNKS; ++c) {
        sX[buf ^ 1][sidx[c]] = rx[c];
        sW[buf ^ 1][sidx[c]] = rw[c];
      }
    }
    __syncthreads();
  }

  // Epilogue.  acc[i][j] register r holds Y[m][n] with
  //   m = m0 + wm + j*32 + lane%32
  //   n = n0 + wn + i*32 + 8*(r/4) + 4*(lane/32) + r%4.
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int m = m0 + wm + j * 32 + l32;
    if (m >= M) continue;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = n0 + wn + i * 32 + g * 8 + lhi * 4;
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

}  // namespace

hipError_t launch_linear(const uint16_t* X, const uint16_t* W, const float* bias, const uint16_t* R,
                         uint16_t* Y, int64_t M, int N, int K, int epi, hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  const int tiles_n = N / BN;
  const int64_t tiles_m = (M + BM - 1) / BM;
  const dim3 grid((unsigned)(tiles_m * tiles_n));
  const dim3 block(THREADS);
  switch (epi) {
    case EPI_BIAS:
      hipLaunchKernelGGL(linear_bf16_kernel<EPI_BIAS>, grid, block, 0, stream, X, W, bias, R, Y,
                         (int)M, N, K, tiles_n);
      break;
    case EPI_BIAS_GELU:
      hipLaunchKernelGGL(linear_bf16_kernel<EPI_BIAS_GELU>, grid, block, 0, stream, X, W, bias, R,
                         Y, (int)M, N, K, tiles_n);
      break;
    default:
      hipLaunchKernelGGL(linear_bf16_kernel<EPI_BIAS_RESIDUAL>, grid, block, 0, stream, X, W, bias,
                         R, Y, (int)M, N, K, tiles_n);
      break;
  }
  return hipGetLastError();
}

}  // namespace surge
