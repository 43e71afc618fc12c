// Projection GEMMs of the DiT block: tile-configuration table, planner and
// dispatch for the bf16 MFMA kernel of gemm_tile.h, plus a plain LDS-tiled
// fp32 kernel for the float32 parity mode.
#include "gemm_tile.h"

namespace wam {

namespace {

using gemm::launch_tile;

// ---------------------------------------------------------------- configs
struct TileCfg {
  int bm, bn, wgm, wgn, st, bk;
};
// index: tile rows x cols, waves (rows x cols), LDS stages, K per stage
constexpr TileCfg kCfgs[] = {
    {64, 64, 2, 2, 4, 32},    // 0
    {64, 128, 2, 2, 4, 32},   // 1
    {128, 64, 2, 2, 4, 32},   // 2
    {128, 128, 2, 2, 4, 32},  // 3
    {256, 256, 2, 4, 4, 32},  // 4
    {256, 256, 4, 2, 4, 32},  // 5
    {256, 128, 2, 4, 4, 32},  // 6
    {128, 256, 2, 4, 4, 32},  // 7
    {128, 128, 2, 4, 4, 32},  // 8
    {64, 256, 1, 4, 4, 32},   // 9
    {64, 64, 2, 2, 8, 32},    // 10
    {64, 128, 2, 2, 8, 32},   // 11
    {128, 64, 2, 2, 8, 32},   // 12
    {64, 64, 2, 2, 12, 32},   // 13
    {128, 128, 2, 2, 8, 32},  // 14
    {64, 64, 2, 2, 4, 128},   // 15
    {64, 128, 2, 2, 3, 128},  // 16
    {128, 64, 2, 2, 3, 128},  // 17
    {64, 64, 2, 2, 4, 64},    // 18
    {64, 128, 2, 2, 4, 64},   // 19
    {128, 128, 2, 4, 4, 64},  // 20
    {256, 256, 4, 2, 2, 64},  // 21
    {256, 256, 2, 4, 2, 64},  // 22
    {128, 128, 2, 2, 4, 64},  // 23
    {192, 256, 2, 4, 2, 64},  // 24
    {320, 256, 2, 4, 2, 64},  // 25
    {64, 64, 4, 1, 4, 32},    // 26 (QKV outputs of 64 mod 128 columns: odd head counts)
    {320, 128, 4, 2, 2, 64},  // 27
};
constexpr int kNumCfgs = sizeof(kCfgs) / sizeof(kCfgs[0]);

template <int C, int ROLE>
hipError_t launch_c(const GemmArgs& a, int splits, hipStream_t s) {
  constexpr TileCfg t = kCfgs[C];
  return launch_tile<t.bm, t.bn, t.wgm, t.wgn, t.st, t.bk, ROLE>(a, splits, s);
}

template <int ROLE>
hipError_t launch_role(const GemmArgs& a, int cfg, int splits, hipStream_t s) {
  switch (cfg) {
    case 0: return launch_c<0, ROLE>(a, splits, s);
    case 1: return launch_c<1, ROLE>(a, splits, s);
    case 2: return launch_c<2, ROLE>(a, splits, s);
    case 3: return launch_c<3, ROLE>(a, splits, s);
    case 4: return launch_c<4, ROLE>(a, splits, s);
    case 5: return launch_c<5, ROLE>(a, splits, s);
    case 6: return launch_c<6, ROLE>(a, splits, s);
    case 7: return launch_c<7, ROLE>(a, splits, s);
    case 8: return launch_c<8, ROLE>(a, splits, s);
    case 9: return launch_c<9, ROLE>(a, splits, s);
    case 10: return launch_c<10, ROLE>(a, splits, s);
    case 11: return launch_c<11, ROLE>(a, splits, s);
    case 12: return launch_c<12, ROLE>(a, splits, s);
    case 13: return launch_c<13, ROLE>(a, splits, s);
    case 14: return launch_c<14, ROLE>(a, splits, s);
    case 15: return launch_c<15, ROLE>(a, splits, s);
    case 16: return launch_c<16, ROLE>(a, splits, s);
    case 17: return launch_c<17, ROLE>(a, splits, s);
    case 18: return launch_c<18, ROLE>(a, splits, s);
    case 19: return launch_c<19, ROLE>(a, splits, s);
    case 20: return launch_c<20, ROLE>(a, splits, s);
    case 21: return launch_c<21, ROLE>(a, splits, s);
    case 22: return launch_c<22, ROLE>(a, splits, s);
    case 23: return launch_c<23, ROLE>(a, splits, s);
    case 24: return launch_c<24, ROLE>(a, splits, s);
    case 25: return launch_c<25, ROLE>(a, splits, s);
    case 26: return launch_c<26, ROLE>(a, splits, s);
    default: return launch_c<27, ROLE>(a, splits, s);
  }
}

bool qkv_ok(int c) { return (kCfgs[c].bn / kCfgs[c].wgn) % 64 == 0; }

// ---------------------------------------------------------------- fp32
constexpr int kFT = 64, kFK = 16;

template <int EPI>
__device__ __forceinline__ void epi1_f32(const GemmArgs& a, int m, int n, float acc) {
  if (m >= a.M) return;
  const float v = acc + a.bias[n];
  if constexpr (EPI == EPI_GATED_RES) {
    float* h = static_cast<float*>(a.out) + (size_t)m * a.N + n;
    const float nv = *h + a.gate[n] * v;
    *h = nv;
    if (a.copy) a.copy[(size_t)m * a.N + n] = nv;
  } else if constexpr (EPI == EPI_BIAS_GELU) {
    static_cast<float*>(a.out)[(size_t)m * a.N + n] = gelu_tanh_f(v);
  } else {
    static_cast<float*>(a.out)[(size_t)m * a.N + n] = v;
  }
}

template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a) {
  if (a.skip && *a.skip) return;
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
      if (n < a.N) epi1_f32<EPI>(a, m0 + ty * 4 + i, n, acc[i][j]);
    }
}

}  // namespace

int gemm_num_configs() { return kNumCfgs; }

GemmPlan plan_gemm(int M, int N, int K, int epi) {
  // From a sweep of every configuration at the workload shapes.  Large M:
  // tiles of 256 columns over 8 waves, K 64 per stage (two stages), with the
  // row count (192, 256 or 320) that minimises whole rounds of one block per
  // CU times rows per block, weighted by the per-row cost each tile height
  // measured (192-row tiles ~10% dearer per row, 320-row ~3% cheaper).  For
  // example M = 9224, N = 4096 (mid MLP-up): 592 blocks of 256 rows take 3
  // rounds, 464 of 320 rows take 2 (98 -> 82 us); M = 9224, N = 1024: 196
  // blocks of 192 rows fill one round that 148 of 256 leave a third idle
  // (97 -> 83 us).  256 rows with K 32 per stage (four stages) for outputs of
  // 1024 columns or fewer, or K not a multiple of 64.  Small M (under a few
  // blocks per CU): 64x64 tiles with K 64 per stage, 64x128 for the QKV
  // epilogue (whole heads per wave), 128x128 over 8 waves for wide, short-K
  // outputs; a K split only for grids under half a block per CU.
  GemmPlan p{0, 1};
  if (M >= 2048 && N % 256 == 0) {
    // outputs of at most 1024 columns whose 320x128 tiles fill one round
    // of 192-256 blocks (the mid model's attention output and MLP-down,
    // N = 1024: 232 blocks, against 196 of 192x256 that leave 60 CUs idle;
    // 34.4 -> 31.8 and 97.4 -> 89.0 us)
    const long b320x128 = (long)((M + 319) / 320) * (N / 128);
    if (K % 64 == 0 && N <= 1024 && b320x128 >= 192 && b320x128 <= 256) {
      p.cfg = 27;
      return p;
    }
    if (K % 64 == 0) {
      const long cols = N / 256;
      auto cost = [&](int bm, double per_row) {
        const long blocks = (M + bm - 1) / bm * cols;
        return (double)((blocks + 255) / 256) * bm * per_row;
      };
      const double c192 = cost(192, 1.10), c256 = cost(256, 1.0), c320 = cost(320, 0.97);
      if (c192 < c256 && c192 <= c320) {
        p.cfg = 24;
        return p;
      }
      if (c320 < c256) {
        p.cfg = 25;
        return p;
      }
    }
    if (N > 1024 && K % 64 == 0) p.cfg = 22;
    else p.cfg = N >= 3072 ? 5 : 4;
    return p;
  }
  if (epi == EPI_QKV) {
    // whole heads per wave: 64 columns per wave; an odd head count leaves
    // N = 192 H a multiple of 64 only, which takes one wave column of 64
    p.cfg = N % 128 != 0 ? 26 : K % 64 == 0 ? 19 : 1;
    return p;
  }
  if (N >= 2048 && N % 128 == 0 && K <= 1024) {
    p.cfg = 8;
    return p;
  }
  const long blocks = (long)((M + 63) / 64) * (N / 64);
  if (K % 64 == 0 && blocks >= 128) {
    p.cfg = 18;
    return p;
  }
  while (blocks * p.splits < 128 && K / (p.splits * 2) >= 768 && K % (gemm::kBK * p.splits * 2) == 0 &&
         p.splits < 8)
    p.splits *= 2;
  return p;
}

size_t gemm_partial_floats(int M, int N, int K, int epi) {
  const GemmPlan p = plan_gemm(M, N, K, epi);
  return p.splits > 1 ? (size_t)p.splits * M * N : 0;
}

hipError_t launch_gemm_cfg(const GemmArgs& a, int cfg, int splits, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (cfg < 0 || cfg >= kNumCfgs || splits < 1) return hipErrorInvalidValue;
  if (a.K % (kCfgs[cfg].bk * splits) || a.N % kCfgs[cfg].bn || a.N % 4) return hipErrorInvalidValue;
  if (splits > 1 && (a.epi == EPI_QKV || !a.partial)) return hipErrorInvalidValue;
  if (a.epi == EPI_QKV && !qkv_ok(cfg)) return hipErrorInvalidValue;
  switch (a.role) {
    case 0: return launch_role<0>(a, cfg, splits, s);
    case 1: return launch_role<1>(a, cfg, splits, s);
    case 2: return launch_role<2>(a, cfg, splits, s);
    default: return launch_role<3>(a, cfg, splits, s);
  }
}

hipError_t launch_gemm(const GemmArgs& a, bool bf16_mode, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (bf16_mode) {
    const GemmPlan p = plan_gemm(a.M, a.N, a.K, a.epi);
    return launch_gemm_cfg(a, p.cfg, p.splits, s);
  }
  if (a.K % kFK || a.epi == EPI_QKV) return hipErrorInvalidValue;
  dim3 grid((a.N + kFT - 1) / kFT, (a.M + kFT - 1) / kFT);
  switch (a.epi) {
    case EPI_BIAS: launch_k(gemm_f32_kernel<EPI_BIAS>, grid, 256, 0, s, a); break;
    case EPI_BIAS_GELU: launch_k(gemm_f32_kernel<EPI_BIAS_GELU>, grid, 256, 0, s, a); break;
    case EPI_GATED_RES: launch_k(gemm_f32_kernel<EPI_GATED_RES>, grid, 256, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace wam
