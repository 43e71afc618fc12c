// Tiled bf16 MFMA GEMM kernel template (gfx950); instantiated by k_gemm.hip.
//
//   C[M][N] = A[M][K] . W[N][K]^T      (both operands K-contiguous, bf16)
//
// v_mfma_f32_16x16x32_bf16 takes the weight tile as its first operand and the
// activation tile as its second, so accumulator element r of a lane is
// C[m = lane%16][n = 4*(lane/16) + r]: each lane owns four consecutive output
// columns of one row and the epilogue stores 8 (bf16) or 16 (fp32) contiguous
// bytes.  A block of WGM x WGN waves owns a BM x BN tile.
//
// K advances BK (32, 64 or 128) at a time through ST LDS stages.  Each stage
// holds BM activation rows and BN weight rows of 2*BK bytes, filled straight
// from global memory by global_load_lds_dwordx4 (16 bytes per lane, one 1 KiB
// run of LDS per instruction, no register staging): ST-1 stages are in flight
// while one is multiplied.  Inside a row the 16-byte chunks are XOR-swizzled
// ((row >> 1) & 3 for 64-byte rows, row & 7 for longer ones), which keeps the
// ds_read_b128 operand reads (16 rows x one chunk per 16 lanes) free of bank
// conflicts; the loads pick their global chunk so that the LDS image comes out
// swizzled.  A deeper stage gives each wave BK/32 MFMA k-steps per barrier,
// which is what short tiles (small M) need.  The compiler cannot follow
// the LDS writes of these loads, so the loop waits on vmcnt itself and uses a
// bare s_barrier (a workgroup fence would drain every load in flight).
// Blocks are renumbered so that each XCD (dispatch is round-robin over 8 XCDs)
// gets a contiguous run of a grouped tile order and shares A rows / W columns
// in its own L2.  With SPLIT, gridDim.z splits K: every split stores an fp32
// partial tile and a second pass sums the partials in split order
// (deterministic) and applies the epilogue.
#pragma once

#include "wam_internal.h"

namespace wam {
namespace gemm {

constexpr int kBK = 32;    // K per MFMA step (and the smallest stage depth)
constexpr int kGroupM = 8;
constexpr int kXcd = 8;

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void global_void;

// s_waitcnt immediate (gfx9 layout: vmcnt bits 3:0 and 15:14, expcnt 6:4,
// lgkmcnt 11:8): at most n vector-memory operations outstanding, no LDS or
// scalar-memory operation outstanding
constexpr int waitcnt_vm_lgkm0(int n) { return (n & 0xf) | ((n >> 4) << 14) | (0x7 << 4); }

// XOR swizzle of the 16-byte chunks of an LDS row of 2*BK bytes
template <int BK>
__device__ __forceinline__ int chunk_swizzle(int row) {
  if constexpr (BK == 32) return (row >> 1) & 3;
  else return row & 7;
}

// compiler-only memory barrier: keeps LDS and global accesses on their side
__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

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
    if (a.copy) *reinterpret_cast<float4*>(a.copy + (size_t)m * a.N + n) = hv;
  } else if constexpr (EPI == EPI_BIAS_GELU) {
    store_bf16x4(static_cast<bf16*>(a.out) + (size_t)m * a.N + n, gelu_tanh_f(v0), gelu_tanh_f(v1),
                 gelu_tanh_f(v2), gelu_tanh_f(v3));
  } else {
    store_bf16x4(static_cast<bf16*>(a.out) + (size_t)m * a.N + n, v0, v1, v2, v3);
  }
}

// Epilogue of one wave's accumulators: acc[j][i] element r is the product at
// row mb + i*16 + lane%16, column nb + j*16 + 4*(lane/16) + r.  SPLIT stores
// the fp32 partial of K split `split`; the others apply the role's epilogue.
template <int EPI, int TN, int TM, bool SPLIT>
__device__ __forceinline__ void store_tile(const GemmArgs& a, const f32x4 (&acc)[TN][TM], int mb, int nb, int lane,
                                           int split) {
  const int lr = lane % 16, lg = lane / 16;
  if constexpr (SPLIT) {
    // fp32 partial tile of this K split; the role's reduce pass finishes it
    float* P = a.partial + (size_t)split * a.M * a.N;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = mb + i * 16 + lr;
      if (m >= a.M) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int n = nb + j * 16 + lg * 4;
        *reinterpret_cast<f32x4*>(P + (size_t)m * a.N + n) = acc[j][i];
      }
    }
  } else if constexpr (EPI == EPI_QKV) {
    const QkvOut& qo = a.qkv;
    const int D = qo.D;
    // per-lane constants hoisted out of the store loop: bias of the lane's
    // columns and the q / k gains of its head dims (d = jj*16 + 4*lg + r)
    f32x4 bias[TN], qg[4], kg[4];
#pragma unroll
    for (int j = 0; j < TN; ++j) bias[j] = *reinterpret_cast<const f32x4*>(a.bias + nb + j * 16 + lg * 4);
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      qg[jj] = kg[jj] = f32x4{1.f, 1.f, 1.f, 1.f};
      if (qo.qk_norm) {
        qg[jj] = *reinterpret_cast<const f32x4*>(qo.q_g + jj * 16 + lg * 4);
        kg[jj] = *reinterpret_cast<const f32x4*>(qo.k_g + jj * 16 + lg * 4);
      }
      qg[jj] *= kQLog2Scale;  // attention scores come out in log2 units
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = mb + i * 16 + lr;
      const int b = m / qo.T, t = m % qo.T;
#pragma unroll
      for (int hs = 0; hs < TN / 4; ++hs) {
        const int nh = nb + hs * 64;  // first column of this head
        const int sec = nh / D, head = (nh % D) / 64;
        f32x4 v[4];
        float ss = 0.f;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          v[jj] = acc[hs * 4 + jj][i] + bias[hs * 4 + jj];
#pragma unroll
          for (int r = 0; r < 4; ++r) ss += v[jj][r] * v[jj][r];
        }
        if (sec < 2) {
          ss += __shfl_xor(ss, 16, 64);
          ss += __shfl_xor(ss, 32, 64);
          const f32x4* gain = sec == 0 ? qg : kg;
          const float rs = qo.qk_norm ? rsqrtf(ss * (1.0f / 64.0f) + qo.eps) : 1.0f;
          if (m < a.M) {
            bf16* dst = (sec == 0 ? qo.q : qo.k) + (((size_t)b * qo.H + head) * qo.Tpad + t) * 64;
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
              const f32x4 o = v[jj] * rs * gain[jj];
              store_bf16x4(dst + jj * 16 + lg * 4, o[0], o[1], o[2], o[3]);
            }
          }
        } else if (m < a.M) {
          // V^T row d holds the tokens of each 64-key block in vt_key_pos order
          bf16* dst = qo.vt + ((size_t)b * qo.H + head) * 64 * qo.Tpad + (t & ~63) + vt_key_pos(t & 63);
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              dst[(size_t)(jj * 16 + lg * 4 + r) * qo.Tpad] = static_cast<bf16>(v[jj][r]);
        }
      }
    }
  } else {
    // bias (and gate) of this lane's columns once, in registers: the output
    // may alias them as far as the compiler knows, so loads inside the store
    // loop would be repeated and serialised behind every store
    f32x4 bias[TN], gate[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = nb + j * 16 + lg * 4;
      bias[j] = *reinterpret_cast<const f32x4*>(a.bias + n);
      if constexpr (EPI == EPI_GATED_RES) gate[j] = *reinterpret_cast<const f32x4*>(a.gate + n);
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = mb + i * 16 + lr;
      if (m >= a.M) continue;
      if constexpr (EPI == EPI_GATED_RES) {
        // residual stream h += gate * (acc + bias): all loads of the row first;
        // with a copy target the new values are stored there as well
        const size_t off = (size_t)m * a.N + nb + lg * 4;
        f32x4* hrow = reinterpret_cast<f32x4*>(static_cast<float*>(a.out) + off);
        f32x4 hv[TN];
#pragma unroll
        for (int j = 0; j < TN; ++j) hv[j] = hrow[j * 4];
#pragma unroll
        for (int j = 0; j < TN; ++j) hv[j] = hv[j] + gate[j] * (acc[j][i] + bias[j]);
#pragma unroll
        for (int j = 0; j < TN; ++j) hrow[j * 4] = hv[j];
        if (a.copy) {
          f32x4* crow = reinterpret_cast<f32x4*>(a.copy + off);
#pragma unroll
          for (int j = 0; j < TN; ++j) crow[j * 4] = hv[j];
        }
      } else {
        bf16* orow = static_cast<bf16*>(a.out) + (size_t)m * a.N + nb + lg * 4;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const f32x4 v = acc[j][i] + bias[j];
          if constexpr (EPI == EPI_BIAS_GELU)
            store_bf16x4(orow + j * 16, gelu_tanh_f(v[0]), gelu_tanh_f(v[1]), gelu_tanh_f(v[2]), gelu_tanh_f(v[3]));
          else
            store_bf16x4(orow + j * 16, v[0], v[1], v[2], v[3]);
        }
      }
    }
  }
}

template <int BM, int BN, int WGM, int WGN, int ST, int BK, int EPI, int ROLE, bool SPLIT>
__global__ __launch_bounds__(WGM* WGN * 64) void gemm_bf16_kernel(GemmArgs a) {
  constexpr int NW = WGM * WGN;
  constexpr int WM = BM / WGM, WN = BN / WGN;  // wave tile
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int ROWS = BM + BN;                // LDS rows per stage: activations, then weights
  constexpr int CPR = BK / 8;                  // 16-byte chunks per LDS row
  constexpr int RPI = 64 / CPR;                // rows per 1 KiB load instruction
  constexpr int NI = ROWS / RPI;               // load instructions per stage
  constexpr int IPW = NI / NW;                 // ... per wave
  constexpr int KS = BK / kBK;                 // MFMA k-steps per stage
  static_assert(BK == 32 || BK == 64 || BK == 128, "stage depth");
  static_assert(TM >= 1 && TN >= 1, "wave tile too small");
  static_assert(IPW >= 1 && IPW * NW == NI, "stage rows / wave mismatch");
  static_assert(EPI != EPI_QKV || WN % 64 == 0, "QKV epilogue needs whole heads per wave");
  static_assert(ST >= 2 && (ST - 2) * IPW < 64, "stage count");
  if (a.skip && *a.skip) return;

  __shared__ __attribute__((aligned(1024))) bf16 sm[ST][ROWS * BK];

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
    const int per = K / gridDim.z;  // host guarantees divisibility by BK * splits
    kbeg = blockIdx.z * per;
    kend = kbeg + per;
  }
  const int nk = (kend - kbeg) / BK;

  // Load instruction j of this wave fills LDS rows RPI*(wid + NW*j) .. +RPI-1;
  // lane l writes LDS chunk l%CPR of row l/CPR, i.e. global chunk
  // (l%CPR) ^ swizzle.  Activation rows past M read row M-1 (their products
  // reach only output rows that are never stored).
  const bf16* src[IPW];
#pragma unroll
  for (int j = 0; j < IPW; ++j) {
    const int row = RPI * (wid + NW * j) + lane / CPR;
    const int col = ((lane % CPR) ^ chunk_swizzle<BK>(row)) * 8;
    src[j] = row < BM ? A + (size_t)min(m0 + row, a.M - 1) * K + kbeg + col
                      : W + (size_t)(n0 + row - BM) * K + kbeg + col;
  }
  auto issue = [&](auto S, int kt) __attribute__((always_inline)) {
    constexpr int s = decltype(S)::value;
#pragma unroll
    for (int j = 0; j < IPW; ++j)
      __builtin_amdgcn_global_load_lds((const global_void*)(src[j] + kt * BK),
                                       (lds_void*)(&sm[s][(wid + NW * j) * RPI * BK]), 16, 0, 0);
  };

  f32x4 acc[TN][TM];
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int i = 0; i < TM; ++i) acc[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};

  // operand reads: for k-step ks, lane (lr, lg) takes chunk 4*ks + lg of row
  // lr of each 16-row tile (tile row offsets are multiples of 16, so the
  // swizzle depends on lr only)
  const int lr = lane % 16, lg = lane / 16;
  const int sw = chunk_swizzle<BK>(lr);
  const int arow = (wm * WM + lr) * BK;
  const int wrow = (BM + wn * WN + lr) * BK;
  auto compute = [&](auto S) __attribute__((always_inline)) {
    constexpr int s = decltype(S)::value;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int ch = ((4 * ks + lg) ^ sw) * 8;
      bf16x8 af[TM], wf[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) af[i] = *reinterpret_cast<const bf16x8*>(&sm[s][arow + ch + i * 16 * BK]);
#pragma unroll
      for (int j = 0; j < TN; ++j) wf[j] = *reinterpret_cast<const bf16x8*>(&sm[s][wrow + ch + j * 16 * BK]);
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int i = 0; i < TM; ++i)
          acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[j], af[i], acc[j][i], 0, 0, 0);
    }
  };
  // one K step on stage slot J: this wave's loads of stage kt have landed (the
  // ST-2 newer stages may still be in flight) and its LDS reads are done;
  // after the barrier everyone's are, and the slot read in the previous step
  // is free for stage kt+ST-1.  Past the last stage the loads repeat it into
  // slots nobody reads again, which keeps the wait counts uniform.
  auto step = [&](auto J, int kt) __attribute__((always_inline)) {
    constexpr int j = decltype(J)::value;
    __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0((ST - 2) * IPW));
    compiler_fence();
    __builtin_amdgcn_s_barrier();
    compiler_fence();
    issue(std::integral_constant<int, (j + ST - 1) % ST>{}, min(kt + ST - 1, nk - 1));
    // the loads must leave before the MFMAs: left to itself the scheduler
    // sinks them below the compute, next to the wait at the top of the next
    // step, which exposes their whole latency every stage
    __builtin_amdgcn_sched_barrier(0);
    compute(J);
  };

  static_for<ST - 1>([&](auto P) __attribute__((always_inline)) { issue(P, min((int)decltype(P)::value, nk - 1)); });
  const int nfull = nk / ST * ST;
  for (int kt0 = 0; kt0 < nfull; kt0 += ST)
    static_for<ST>([&](auto J) __attribute__((always_inline)) { step(J, kt0 + decltype(J)::value); });
  static_for<ST - 1>([&](auto J) __attribute__((always_inline)) {
    const int kt = nfull + decltype(J)::value;
    if (kt < nk) step(J, kt);
  });
  // no load may still be writing this block's LDS when the block retires
  __builtin_amdgcn_s_waitcnt(0);

  store_tile<EPI, TN, TM, SPLIT>(a, acc, m0 + wm * WM, n0 + wn * WN, lane, blockIdx.z);
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

template <int BM, int BN, int WGM, int WGN, int ST, int BK, int ROLE>
hipError_t launch_tile(const GemmArgs& a, int splits, hipStream_t s) {
  const int blocks = ((a.M + BM - 1) / BM) * (a.N / BN);
  constexpr int NT = WGM * WGN * 64;
  if (splits > 1) {
    dim3 grid(blocks, 1, splits);
    launch_k(gemm_bf16_kernel<BM, BN, WGM, WGN, ST, BK, EPI_BIAS, ROLE, true>, grid, NT, 0, s, a);
    const int64_t n4 = (int64_t)a.M * a.N / 4;
    const unsigned rb = (unsigned)((n4 + 255) / 256);
    switch (a.epi) {
      case EPI_BIAS: launch_k(gemm_splitk_reduce_kernel<EPI_BIAS, ROLE>, rb, 256, 0, s, a, splits); break;
      case EPI_BIAS_GELU: launch_k(gemm_splitk_reduce_kernel<EPI_BIAS_GELU, ROLE>, rb, 256, 0, s, a, splits); break;
      case EPI_GATED_RES: launch_k(gemm_splitk_reduce_kernel<EPI_GATED_RES, ROLE>, rb, 256, 0, s, a, splits); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  switch (a.epi) {
    case EPI_BIAS:
      launch_k(gemm_bf16_kernel<BM, BN, WGM, WGN, ST, BK, EPI_BIAS, ROLE, false>, blocks, NT, 0, s, a);
      break;
    case EPI_BIAS_GELU:
      launch_k(gemm_bf16_kernel<BM, BN, WGM, WGN, ST, BK, EPI_BIAS_GELU, ROLE, false>, blocks, NT, 0, s, a);
      break;
    case EPI_GATED_RES:
      launch_k(gemm_bf16_kernel<BM, BN, WGM, WGN, ST, BK, EPI_GATED_RES, ROLE, false>, blocks, NT, 0, s, a);
      break;
    case EPI_QKV:
      if constexpr ((BN / WGN) % 64 == 0) {
        launch_k(gemm_bf16_kernel<BM, BN, WGM, WGN, ST, BK, EPI_QKV, ROLE, false>, blocks, NT, 0, s, a);
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
