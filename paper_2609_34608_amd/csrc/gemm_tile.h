// Tiled bf16 MFMA GEMM kernel template (gfx950); instantiated by k_gemm.hip.
//
//   C[M][N] = A[M][K] . W[N][K]^T      (both operands K-contiguous, bf16)
//
// v_mfma_f32_16x16x32_bf16 takes the weight tile as its first operand and the
// activation tile as its second, so accumulator element r of a lane is
// C[m = lane%16][n = 4*(lane/16) + r]: each lane owns four consecutive output
// columns of one row and the epilogue stores 8 (bf16) or 16 (fp32) contiguous
// bytes.  A block of WGM x WGN waves owns a BM x BN tile.  K advances 64 at a
// time through a double-buffered LDS ring whose rows are padded to 72 bf16 (the
// 16 rows one MFMA operand read touches fall in distinct banks).  The ring is
// fed from registers that hold the next PF K tiles: loads for tile kt+PF are
// issued while tile kt is multiplied, so PF tiles are in flight per block (the
// loop is unrolled by PF so that every register slot is static).  Blocks are
// renumbered so that each XCD (dispatch is round-robin over 8 XCDs) gets a
// contiguous run of a grouped tile order and shares A rows / W columns in its
// own L2.  With SPLIT, gridDim.z splits K: every split stores an fp32 partial
// tile and a second pass sums the partials in split order (deterministic) and
// applies the epilogue.  (A single-kernel variant in which the last-arriving
// block of a tile does that sum needs agent-scope release/acquire fences, which
// write back and invalidate the XCD L2s in every block: measured 4-5x slower.)
#pragma once

#include "wam_internal.h"

namespace wam {
namespace gemm {

constexpr int kBK = 64;
constexpr int kPad = 8;
constexpr int kLds = kBK + kPad;  // bf16 elements per LDS row
constexpr int kGroupM = 8;
constexpr int kXcd = 8;

__device__ __forceinline__ void tile_coords(int bid, int nblocks, int tiles_m, int tiles_n, int& tm,
                                            int& tn) {
  const int per = nblocks / kXcd, rem = nblocks % kXcd;
  const int x = bid % kXcd, idx = bid / kXcd;
  const int logical = x * per + min(x, rem) + idx;
  const int width = kGroupM * tiles_n;
  const int group = logical / width;
  const int first_m = group * kGroupM;
  const int gsz = min(tiles_m - first_m, kGroupM);
  const int in = logical % width;
  tm = first_m + in % gsz;
  tn = in / gsz;
}

__device__ __forceinline__ void store_bf16x4(bf16* p, float a, float b, float c, float d) {
  bf16x4 v = {static_cast<bf16>(a), static_cast<bf16>(b), static_cast<bf16>(c), static_cast<bf16>(d)};
  *reinterpret_cast<bf16x4*>(p) = v;
}

// Elementwise epilogue on four consecutive columns n..n+3 of row m.
template <int EPI>
__device__ __forceinline__ void epi4(const GemmArgs& a, int m, int n, float v0, float v1, float v2, float v3) {
  const float4 b = *reinterpret_cast<const float4*>(a.bias + n);
  v0 += b.x; v1 += b.y; v2 += b.z; v3 += b.w;
  if constexpr (EPI == EPI_GATED_RES) {
    const float4 g = *reinterpret_cast<const float4*>(a.gate + n);
    float4* h = reinterpret_cast<float4*>(static_cast<float*>(a.out) + (size_t)m * a.N + n);
    float4 hv = *h;
    hv.x += g.x * v0; hv.y += g.y * v1; hv.z += g.z * v2; hv.w += g.w * v3;
    *h = hv;
  } else if constexpr (EPI == EPI_BIAS_GELU) {
    store_bf16x4(static_cast<bf16*>(a.out) + (size_t)m * a.N + n, gelu_tanh_f(v0), gelu_tanh_f(v1),
                 gelu_tanh_f(v2), gelu_tanh_f(v3));
  } else {
    store_bf16x4(static_cast<bf16*>(a.out) + (size_t)m * a.N + n, v0, v1, v2, v3);
  }
}

template <int BM, int BN, int WGM, int WGN, int PF, int EPI, int ROLE, bool SPLIT>
__global__ __launch_bounds__(WGM* WGN * 64) void gemm_bf16_kernel(GemmArgs a) {
  constexpr int NT = WGM * WGN * 64;
  constexpr int WM = BM / WGM, WN = BN / WGN;  // wave tile
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int ACH = BM * (kBK / 8) / NT;  // 16-byte chunks per thread per K tile
  constexpr int BCH = BN * (kBK / 8) / NT;
  static_assert(TM >= 1 && TN >= 1, "wave tile too small");
  static_assert(ACH >= 1 && BCH >= 1 && ACH * NT == BM * 8 && BCH * NT == BN * 8, "tile / thread mismatch");
  static_assert(EPI != EPI_QKV || WN % 64 == 0, "QKV epilogue needs whole heads per wave");
  static_assert(PF >= 1, "prefetch depth");
  if (a.skip && *a.skip) return;

  __shared__ __attribute__((aligned(16))) bf16 As[2][BM][kLds];
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][BN][kLds];

  const int tiles_m = (a.M + BM - 1) / BM, tiles_n = a.N / BN;
  int tm, tn;
  tile_coords(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid % 64, wid = tid / 64;
  const int wm = wid / WGN, wn = wid % WGN;
  const bf16* A = static_cast<const bf16*>(a.A);
  const bf16* W = static_cast<const bf16*>(a.W);
  const int K = a.K;
  int kbeg = 0, kend = K;
  if constexpr (SPLIT) {
    const int per = K / gridDim.z;  // host guarantees divisibility by 64 * splits
    kbeg = blockIdx.z * per;
    kend = kbeg + per;
  }
  const int nk = (kend - kbeg) / kBK;

  // per-thread global offsets; tile rows past M read row M-1 instead (their
  // products only reach output rows that are never stored, and loading
  // unmasked keeps the prefetch free of waits on its own data)
  const bf16* pa[ACH];
#pragma unroll
  for (int i = 0; i < ACH; ++i) {
    const int c = tid + NT * i, row = c >> 3, col = (c & 7) * 8;
    pa[i] = A + (size_t)min(m0 + row, a.M - 1) * K + kbeg + col;
  }
  const bf16* pw[BCH];
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    const int c = tid + NT * i, row = c >> 3, col = (c & 7) * 8;
    pw[i] = W + (size_t)(n0 + row) * K + kbeg + col;
  }

  u32x4 ra[PF][ACH], rb[PF][BCH];
  auto gload = [&](auto S, int kt) __attribute__((always_inline)) {
    constexpr int slot = decltype(S)::value;
#pragma unroll
    for (int i = 0; i < ACH; ++i) ra[slot][i] = *reinterpret_cast<const u32x4*>(pa[i] + kt * kBK);
#pragma unroll
    for (int i = 0; i < BCH; ++i) rb[slot][i] = *reinterpret_cast<const u32x4*>(pw[i] + kt * kBK);
  };
  auto sstore = [&](auto S, int buf) __attribute__((always_inline)) {
    constexpr int slot = decltype(S)::value;
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int c = tid + NT * i, row = c >> 3, col = (c & 7) * 8;
      *reinterpret_cast<u32x4*>(&As[buf][row][col]) = ra[slot][i];
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int c = tid + NT * i, row = c >> 3, col = (c & 7) * 8;
      *reinterpret_cast<u32x4*>(&Bs[buf][row][col]) = rb[slot][i];
    }
  };

  f32x4 acc[TN][TM];
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int i = 0; i < TM; ++i) acc[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int lr = lane % 16, lg = lane / 16, lk = lg * 8;
  auto compute = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < kBK / 32; ++ks) {
      bf16x8 af[TM], wf[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(&As[buf][wm * WM + i * 16 + lr][ks * 32 + lk]);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        wf[j] = *reinterpret_cast<const bf16x8*>(&Bs[buf][wn * WN + j * 16 + lr][ks * 32 + lk]);
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int i = 0; i < TM; ++i)
          acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[j], af[i], acc[j][i], 0, 0, 0);
    }
  };

  // prologue: tiles 0 .. PF-1 in flight, tile 0 into LDS
  static_for<PF>([&](auto P) __attribute__((always_inline)) {
    if (decltype(P)::value < nk) gload(P, decltype(P)::value);
  });
  sstore(std::integral_constant<int, 0>{}, 0);
  __syncthreads();
  // steady state, unrolled by PF: register slot of tile t is t % PF, LDS
  // buffer t % 2.  Full groups of PF tiles run branch-free (the prefetch index
  // is clamped to the last tile, and a store after the last tile lands in the
  // buffer nobody reads again), so the compiler's wait counts stay exact and
  // PF tiles really are in flight; only the last partial group branches.
  const int nfull = nk / PF * PF;
  for (int kt0 = 0; kt0 < nfull; kt0 += PF) {
    static_for<PF>([&](auto J) __attribute__((always_inline)) {
      constexpr int j = decltype(J)::value;
      const int kt = kt0 + j;
      gload(J, min(kt + PF, nk - 1));  // slot j held tile kt, already in LDS
      compute(kt & 1);
      sstore(std::integral_constant<int, (j + 1) % PF>{}, (kt + 1) & 1);
      __syncthreads();
    });
  }
  static_for<PF>([&](auto J) __attribute__((always_inline)) {
    constexpr int j = decltype(J)::value;
    const int kt = nfull + j;
    if (kt < nk) {
      compute(kt & 1);
      if (kt + 1 < nk) sstore(std::integral_constant<int, (j + 1) % PF>{}, (kt + 1) & 1);
      __syncthreads();
    }
  });

  // accumulator (j,i) element r: row m = i*16 + lane%16, column n = j*16 + 4*(lane/16) + r
  if constexpr (SPLIT) {
    // fp32 partial tile of this K split; the role's reduce pass finishes it
    float* P = a.partial + (size_t)blockIdx.z * a.M * a.N;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = m0 + wm * WM + i * 16 + lr;
      if (m >= a.M) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int n = n0 + wn * WN + j * 16 + lg * 4;
        *reinterpret_cast<f32x4*>(P + (size_t)m * a.N + n) = acc[j][i];
      }
    }
  } else if constexpr (EPI == EPI_QKV) {
    const QkvOut& qo = a.qkv;
    const int D = qo.D;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = m0 + wm * WM + i * 16 + lr;
      const int b = m / qo.T, t = m % qo.T;
#pragma unroll
      for (int hs = 0; hs < WN / 64; ++hs) {
        const int nh = n0 + wn * WN + hs * 64;  // first column of this head
        const int sec = nh / D, head = (nh % D) / 64;
        float v[4][4];
        float ss = 0.f;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int n = nh + jj * 16 + lg * 4;
          const float4 bb = *reinterpret_cast<const float4*>(a.bias + n);
          v[jj][0] = acc[hs * 4 + jj][i][0] + bb.x;
          v[jj][1] = acc[hs * 4 + jj][i][1] + bb.y;
          v[jj][2] = acc[hs * 4 + jj][i][2] + bb.z;
          v[jj][3] = acc[hs * 4 + jj][i][3] + bb.w;
#pragma unroll
          for (int r = 0; r < 4; ++r) ss += v[jj][r] * v[jj][r];
        }
        if (sec < 2) {
          ss += __shfl_xor(ss, 16, 64);
          ss += __shfl_xor(ss, 32, 64);
          const float* gain = sec == 0 ? qo.q_g : qo.k_g;
          const float rs = qo.qk_norm ? rsqrtf(ss * (1.0f / 64.0f) + qo.eps) : 1.0f;
          if (m < a.M) {
            bf16* dst = (sec == 0 ? qo.q : qo.k) + (((size_t)b * qo.H + head) * qo.Tpad + t) * 64;
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
              const int d = jj * 16 + lg * 4;
              float4 gg = make_float4(1.f, 1.f, 1.f, 1.f);
              if (qo.qk_norm) gg = *reinterpret_cast<const float4*>(gain + d);
              store_bf16x4(dst + d, v[jj][0] * rs * gg.x, v[jj][1] * rs * gg.y, v[jj][2] * rs * gg.z,
                           v[jj][3] * rs * gg.w);
            }
          }
        } else if (m < a.M) {
          bf16* dst = qo.vt + ((size_t)b * qo.H + head) * 64 * qo.Tpad + t;
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              dst[(size_t)(jj * 16 + lg * 4 + r) * qo.Tpad] = static_cast<bf16>(v[jj][r]);
        }
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = m0 + wm * WM + i * 16 + lr;
      if (m >= a.M) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int n = n0 + wn * WN + j * 16 + lg * 4;
        epi4<EPI>(a, m, n, acc[j][i][0], acc[j][i][1], acc[j][i][2], acc[j][i][3]);
      }
    }
  }
}

// Split-K second pass: sum the partials in split order, then the epilogue.
template <int EPI, int ROLE>
__global__ __launch_bounds__(256) void gemm_splitk_reduce_kernel(GemmArgs a, int splits) {
  if (a.skip && *a.skip) return;
  const int64_t i4 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t n4 = (int64_t)a.M * a.N / 4;
  if (i4 >= n4) return;
  const int m = (int)((i4 * 4) / a.N), n = (int)((i4 * 4) % a.N);
  f32x4 sum = reinterpret_cast<const f32x4*>(a.partial)[i4];
  for (int z = 1; z < splits; ++z) sum += reinterpret_cast<const f32x4*>(a.partial + (size_t)z * a.M * a.N)[i4];
  epi4<EPI>(a, m, n, sum[0], sum[1], sum[2], sum[3]);
}

template <int BM, int BN, int WGM, int WGN, int PF, int ROLE>
hipError_t launch_tile(const GemmArgs& a, int splits, hipStream_t s) {
  const int blocks = ((a.M + BM - 1) / BM) * (a.N / BN);
  constexpr int NT = WGM * WGN * 64;
  if (splits > 1) {
    dim3 grid(blocks, 1, splits);
    gemm_bf16_kernel<BM, BN, WGM, WGN, PF, EPI_BIAS, ROLE, true><<<grid, NT, 0, s>>>(a);
    const int64_t n4 = (int64_t)a.M * a.N / 4;
    const unsigned rb = (unsigned)((n4 + 255) / 256);
    switch (a.epi) {
      case EPI_BIAS: gemm_splitk_reduce_kernel<EPI_BIAS, ROLE><<<rb, 256, 0, s>>>(a, splits); break;
      case EPI_BIAS_GELU: gemm_splitk_reduce_kernel<EPI_BIAS_GELU, ROLE><<<rb, 256, 0, s>>>(a, splits); break;
      case EPI_GATED_RES: gemm_splitk_reduce_kernel<EPI_GATED_RES, ROLE><<<rb, 256, 0, s>>>(a, splits); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  switch (a.epi) {
    case EPI_BIAS:
      gemm_bf16_kernel<BM, BN, WGM, WGN, PF, EPI_BIAS, ROLE, false><<<blocks, NT, 0, s>>>(a);
      break;
    case EPI_BIAS_GELU:
      gemm_bf16_kernel<BM, BN, WGM, WGN, PF, EPI_BIAS_GELU, ROLE, false><<<blocks, NT, 0, s>>>(a);
      break;
    case EPI_GATED_RES:
      gemm_bf16_kernel<BM, BN, WGM, WGN, PF, EPI_GATED_RES, ROLE, false><<<blocks, NT, 0, s>>>(a);
      break;
    case EPI_QKV:
      if constexpr ((BN / WGN) % 64 == 0) {
        gemm_bf16_kernel<BM, BN, WGM, WGN, PF, EPI_QKV, ROLE, false><<<blocks, NT, 0, s>>>(a);
      } else {
        return hipErrorInvalidValue;
      }
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace gemm
}  // namespace wam
