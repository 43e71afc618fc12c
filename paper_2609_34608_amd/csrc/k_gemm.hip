// Projection GEMMs of the DiT block with fused epilogues (gfx950).
//
//   C[M][N] = A[M][K] . W[N][K]^T      (both operands K-contiguous)
//
// bf16 path: v_mfma_f32_16x16x32_bf16, 256 threads = 4 waves in a 2x2 grid,
// block tile BM x BN x 64, LDS double buffer filled from a register prefetch
// of the next K tile, padded LDS rows (64+8 bf16) so that the 16 lanes of an
// MFMA operand read hit distinct banks.  Blocks are renumbered so that each
// XCD (blocks are dispatched round-robin over the 8 XCDs) gets a contiguous
// run of a grouped tile order and shares A rows / W columns in its own L2.
//
// fp32 path: plain LDS-tiled FMA kernel (used by the float32 parity mode).
#include "wam_internal.h"

namespace wam {

namespace {

constexpr int kBK = 64;
constexpr int kPad = 8;
constexpr int kLds = kBK + kPad;  // bf16 elements per LDS row
constexpr int kThreads = 256;
constexpr int kGroupM = 8;
constexpr int kXcd = 8;

__device__ __forceinline__ void tile_coords(int bid, int nblocks, int tiles_m, int tiles_n,
                                            int& tm, int& tn) {
  // XCD-contiguous renumbering (bijective for round-robin dispatch).
  const int per = nblocks / kXcd, rem = nblocks % kXcd;
  const int x = bid % kXcd, idx = bid / kXcd;
  const int logical = x * per + min(x, rem) + idx;
  // grouped order: kGroupM tile rows swept column by column
  const int width = kGroupM * tiles_n;
  const int group = logical / width;
  const int first_m = group * kGroupM;
  const int gsz = min(tiles_m - first_m, kGroupM);
  const int in = logical % width;
  tm = first_m + in % gsz;
  tn = in / gsz;
}

template <int EPI, typename TOut>
__device__ __forceinline__ void epilogue_store(const GemmArgs& a, int m, int n, float acc) {
  if (m >= a.M) return;
  const float v = acc + a.bias[n];
  if constexpr (EPI == EPI_GATED_RES) {
    float* h = static_cast<float*>(a.out) + (size_t)m * a.N + n;
    *h += a.gate[n] * v;
  } else if constexpr (EPI == EPI_BIAS_GELU) {
    static_cast<TOut*>(a.out)[(size_t)m * a.N + n] = from_f32<TOut>(gelu_tanh_f(v));
  } else {
    static_cast<TOut*>(a.out)[(size_t)m * a.N + n] = from_f32<TOut>(v);
  }
}

template <int BM, int BN, int EPI>
__global__ __launch_bounds__(kThreads) void gemm_bf16_kernel(GemmArgs a) {
  constexpr int WM = BM / 2, WN = BN / 2;  // wave tile
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int ACH = BM * (kBK / 8) / kThreads;  // 16-byte chunks per thread
  constexpr int BCH = BN * (kBK / 8) / kThreads;
  static_assert(ACH >= 1 && BCH >= 1, "tile too small");

  __shared__ __attribute__((aligned(16))) bf16 As[2][BM][kLds];
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][BN][kLds];

  const int tiles_m = (a.M + BM - 1) / BM, tiles_n = a.N / BN;
  int tm, tn;
  tile_coords(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid % kWave, wid = tid / kWave;
  const int wm = wid / 2, wn = wid % 2;
  const bf16* A = static_cast<const bf16*>(a.A);
  const bf16* W = static_cast<const bf16*>(a.W);
  const int K = a.K;

  uint4 ra[ACH], rb[BCH];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int c = tid + kThreads * i, row = c >> 3, col = (c & 7) * 8;
      const int m = m0 + row;
      ra[i] = m < a.M ? *reinterpret_cast<const uint4*>(A + (size_t)m * K + k0 + col)
                      : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int c = tid + kThreads * i, row = c >> 3, col = (c & 7) * 8;
      rb[i] = *reinterpret_cast<const uint4*>(W + (size_t)(n0 + row) * K + k0 + col);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int c = tid + kThreads * i, row = c >> 3, col = (c & 7) * 8;
      *reinterpret_cast<uint4*>(&As[buf][row][col]) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int c = tid + kThreads * i, row = c >> 3, col = (c & 7) * 8;
      *reinterpret_cast<uint4*>(&Bs[buf][row][col]) = rb[i];
    }
  };

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = K / kBK;
  gload(0);
  sstore(0);
  __syncthreads();
  const int lr = lane % 16, lk = (lane / 16) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * kBK);
#pragma unroll
    for (int ks = 0; ks < kBK / 32; ++ks) {
      bf16x8 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(&As[buf][wm * WM + i * 16 + lr][ks * 32 + lk]);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8*>(&Bs[buf][wn * WN + j * 16 + lr][ks * 32 + lk]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }

  // accumulator (i,j) element r: row i*16 + 4*(lane/16) + r, column j*16 + lane%16
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm * WM + i * 16 + (lane / 16) * 4 + r;
        const int n = n0 + wn * WN + j * 16 + lr;
        epilogue_store<EPI, bf16>(a, m, n, acc[i][j][r]);
      }
}

// ---------------------------------------------------------------- fp32
constexpr int kFT = 64, kFK = 16;

template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a) {
  __shared__ float As[kFK][kFT + 4];
  __shared__ float Bs[kFK][kFT + 4];
  const int m0 = blockIdx.y * kFT, n0 = blockIdx.x * kFT;
  const int tid = threadIdx.x, ty = tid / 16, tx = tid % 16;
  const float* A = static_cast<const float*>(a.A);
  const float* W = static_cast<const float*>(a.W);
  float acc[4][4] = {};
  const int lrow = tid / 4, lk = (tid % 4) * 4;
  for (int k0 = 0; k0 < a.K; k0 += kFK) {
    {
      const int m = m0 + lrow;
      float4 v = m < a.M ? *reinterpret_cast<const float4*>(A + (size_t)m * a.K + k0 + lk)
                         : make_float4(0.f, 0.f, 0.f, 0.f);
      As[lk + 0][lrow] = v.x; As[lk + 1][lrow] = v.y; As[lk + 2][lrow] = v.z; As[lk + 3][lrow] = v.w;
      const int n = n0 + lrow;
      float4 w = n < a.N ? *reinterpret_cast<const float4*>(W + (size_t)n * a.K + k0 + lk)
                         : make_float4(0.f, 0.f, 0.f, 0.f);
      Bs[lk + 0][lrow] = w.x; Bs[lk + 1][lrow] = w.y; Bs[lk + 2][lrow] = w.z; Bs[lk + 3][lrow] = w.w;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kFK; ++k) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[k][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = Bs[k][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += av[i] * bv[j];
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n < a.N) epilogue_store<EPI, float>(a, m0 + ty * 4 + i, n, acc[i][j]);
    }
}

template <int BM, int BN>
hipError_t launch_bf16_tile(const GemmArgs& a, hipStream_t s) {
  const int blocks = ((a.M + BM - 1) / BM) * (a.N / BN);
  switch (a.epi) {
    case EPI_BIAS: gemm_bf16_kernel<BM, BN, EPI_BIAS><<<blocks, kThreads, 0, s>>>(a); break;
    case EPI_BIAS_GELU: gemm_bf16_kernel<BM, BN, EPI_BIAS_GELU><<<blocks, kThreads, 0, s>>>(a); break;
    case EPI_GATED_RES: gemm_bf16_kernel<BM, BN, EPI_GATED_RES><<<blocks, kThreads, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& a, bool bf16_mode, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (bf16_mode) {
    if (a.K % kBK || a.N % 64) return hipErrorInvalidValue;
    const long big = (long)((a.M + 127) / 128) * (a.N / 128);
    if (a.N % 128 == 0 && big >= 2L * 256) return launch_bf16_tile<128, 128>(a, s);
    return launch_bf16_tile<64, 64>(a, s);
  }
  if (a.K % kFK) return hipErrorInvalidValue;
  dim3 grid((a.N + kFT - 1) / kFT, (a.M + kFT - 1) / kFT);
  switch (a.epi) {
    case EPI_BIAS: gemm_f32_kernel<EPI_BIAS><<<grid, 256, 0, s>>>(a); break;
    case EPI_BIAS_GELU: gemm_f32_kernel<EPI_BIAS_GELU><<<grid, 256, 0, s>>>(a); break;
    case EPI_GATED_RES: gemm_f32_kernel<EPI_GATED_RES><<<grid, 256, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace wam
