// Bidirectional softmax attention over the joint token sequence (gfx950).
//
// qkv_relayout: [B*T][3D] projection output -> per-head q, k ([B*H][Tpad][dh],
// RMS-normalised with gains when QK-norm is on) and v transposed
// ([B*H][dh][Tpad]).  Pad rows/columns beyond T are never written; the host
// zero-fills them once.
//
// bf16 flash attention (dh = 64): each wave owns 16*QT queries and keeps their
// Q fragments in registers.  Scores are formed transposed, S^T = K Q^T, with
// v_mfma_f32_16x16x32_bf16 so that a lane's accumulators all belong to one
// query column: the online-softmax rescale of O^T = V^T P^T is lane-local and
// the running max needs only two cross-lane steps.  P^T feeds the second MFMA
// straight from registers; the key order inside the 32-key contraction is
// permuted consistently on both operands (a contraction is order-free), so V^T
// is read from LDS as two 8-byte runs per lane.  K and V^T tiles of 64 keys are
// double-buffered in LDS and prefetched through registers.  Softmax runs in
// fp32 with exp2 and a log2(e)/sqrt(dh) pre-scale.
#include <math.h>

#include "wam_internal.h"

namespace wam {

namespace {

// ------------------------------------------------------------- relayout
template <typename T, int DH>
__global__ __launch_bounds__(256) void qkv_relayout_kernel(RelayoutArgs a) {
  if (a.skip && *a.skip) return;
  constexpr int TT = 64;  // tokens per block
  __shared__ float vs[DH][TT + 1];
  const int t0 = blockIdx.x * TT, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid % kWave, wid = tid / kWave;
  const T* qkv = static_cast<const T*>(a.qkv);
  const size_t bh = (size_t)b * a.H + h;
  T* qo = static_cast<T*>(a.q) + bh * a.Tpad * DH;
  T* ko = static_cast<T*>(a.k) + bh * a.Tpad * DH;
  T* vo = static_cast<T*>(a.vt) + bh * DH * a.Tpad;
  // q and k: one wave per token row, lane = feature (DH <= 64)
  for (int tt = wid; tt < TT; tt += 4) {
    const int t = t0 + tt;
    if (t >= a.T) break;
    const T* src = qkv + ((size_t)b * a.T + t) * 3 * a.D + h * DH;
    float qv = lane < DH ? to_f32(src[lane]) : 0.f;
    float kv = lane < DH ? to_f32(src[a.D + lane]) : 0.f;
    const float vv = lane < DH ? to_f32(src[2 * a.D + lane]) : 0.f;
    if (a.qk_norm) {
      const float rq = rsqrtf(wave_sum(qv * qv) / (float)DH + a.eps);
      const float rk = rsqrtf(wave_sum(kv * kv) / (float)DH + a.eps);
      if (lane < DH) {
        qv = qv * rq * a.q_g[lane];
        kv = kv * rk * a.k_g[lane];
      }
    }
    if (lane < DH) {
      qo[(size_t)t * DH + lane] = from_f32<T>(qv);
      ko[(size_t)t * DH + lane] = from_f32<T>(kv);
      vs[lane][tt] = vv;
    }
  }
  __syncthreads();
  // v^T: row d holds tokens t0 .. t0+63 contiguously
  for (int i = tid; i < DH * TT; i += 256) {
    const int d = i / TT, tt = i % TT;
    const int t = t0 + tt;
    if (t < a.T) vo[(size_t)d * a.Tpad + t] = from_f32<T>(vs[d][tt]);
  }
}

// ------------------------------------------------------------- bf16 flash attention
constexpr int kDh = 64;
constexpr int kKB = 64;           // keys per tile
constexpr int kKL = kDh + 8;      // LDS row (K tile): 64 dh + pad
constexpr int kVL = kKB + 8;      // LDS row (V^T tile): 64 keys + pad

template <int QT, int NW, int PF>
__global__ __launch_bounds__(NW * 64) void attn_bf16_kernel(AttnArgs a, float scale_log2) {
  if (a.skip && *a.skip) return;
  constexpr int NT = NW * 64;
  constexpr int QB = NW * QT * 16;  // queries per block
  __shared__ __attribute__((aligned(16))) bf16 Ks[2][kKB][kKL];
  __shared__ __attribute__((aligned(16))) bf16 Vs[2][kDh][kVL];

  const int bh = blockIdx.y;
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, lane = tid % 64, wid = tid / 64;
  const int q0 = blockIdx.x * QB + wid * QT * 16;
  const int g = lane / 16, lr = lane % 16;

  const bf16* Q = static_cast<const bf16*>(a.q) + (size_t)bh * a.Tpad * kDh;
  const bf16* Kg = static_cast<const bf16*>(a.k) + (size_t)bh * a.Tpad * kDh;
  const bf16* Vg = static_cast<const bf16*>(a.vt) + (size_t)bh * kDh * a.Tpad;

  // Q fragments (B operand of S^T = K Q^T): query q0 + qt*16 + lr, dh chunk c
  bf16x8 qf[QT][2];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt)
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int q = q0 + qt * 16 + lr;
      qf[qt][c] = q < a.Tpad ? *reinterpret_cast<const bf16x8*>(Q + (size_t)q * kDh + c * 32 + g * 8)
                             : bf16x8{};
    }

  f32x4 o[4][QT];  // O^T tiles: dh tile x query tile
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) o[d][qt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float mrun[QT], lrun[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    mrun[qt] = -INFINITY;
    lrun[qt] = 0.f;
  }

  // K and V^T tiles of 64 keys: 512 chunks of 16 B each, CH per thread;
  // register slots hold the next PF tiles (slot of tile t is t % PF)
  constexpr int CH = 512 / NT;
  static_assert(CH >= 1 && CH * NT == 512, "tile load split");
  u32x4 rk[PF][CH], rv[PF][CH];
  auto gload = [&](auto S, int k0) __attribute__((always_inline)) {
    constexpr int slot = decltype(S)::value;
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = tid + NT * i, row = c >> 3, col = (c & 7) * 8;
      rk[slot][i] = *reinterpret_cast<const u32x4*>(Kg + (size_t)(k0 + row) * kDh + col);
      rv[slot][i] = *reinterpret_cast<const u32x4*>(Vg + (size_t)row * a.Tpad + k0 + col);
    }
  };
  auto sstore = [&](auto S, int buf) __attribute__((always_inline)) {
    constexpr int slot = decltype(S)::value;
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = tid + NT * i, row = c >> 3, col = (c & 7) * 8;
      *reinterpret_cast<u32x4*>(&Ks[buf][row][col]) = rk[slot][i];
      *reinterpret_cast<u32x4*>(&Vs[buf][row][col]) = rv[slot][i];
    }
  };

  auto block = [&](int buf, int k0, auto MASK) __attribute__((always_inline)) {
    // S^T tiles [key tile kt][query tile qt]
    f32x4 s[4][QT];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      const bf16x8 k0f = *reinterpret_cast<const bf16x8*>(&Ks[buf][kt * 16 + lr][g * 8]);
      const bf16x8 k1f = *reinterpret_cast<const bf16x8*>(&Ks[buf][kt * 16 + lr][32 + g * 8]);
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        f32x4 z = {0.f, 0.f, 0.f, 0.f};
        z = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0f, qf[qt][0], z, 0, 0, 0);
        s[kt][qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1f, qf[qt][1], z, 0, 0, 0);
      }
    }
    // mask keys >= T (key of element r: k0 + kt*16 + 4g + r); only the last
    // key tile can hold such keys, so only its instance carries the mask
    if constexpr (decltype(MASK)::value) {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bool live = k0 + kt * 16 + g * 4 + r < a.T;
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) s[kt][qt][r] = live ? s[kt][qt][r] : -INFINITY;
        }
    }
    // online softmax per query column (lane-local except the max)
    bf16x8 pf[2][QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) mx = fmaxf(mx, s[kt][qt][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mnew = fmaxf(mrun[qt], mx * scale_log2);
      const float corr = __builtin_amdgcn_exp2f(mrun[qt] - mnew);
      mrun[qt] = mnew;
      float ls = 0.f;
      float p[4][4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          p[kt][r] = __builtin_amdgcn_exp2f(s[kt][qt][r] * scale_log2 - mnew);
          ls += p[kt][r];
        }
      lrun[qt] = lrun[qt] * corr + ls;
#pragma unroll
      for (int d = 0; d < 4; ++d) o[d][qt] *= corr;
      // B operand of O^T += V^T P^T for key chunk c: slots 0-3 = key tile 2c,
      // slots 4-7 = key tile 2c+1 (keys 4g+r within each)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        bf16x8 v;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          v[r] = static_cast<bf16>(p[2 * c][r]);
          v[4 + r] = static_cast<bf16>(p[2 * c + 1][r]);
        }
        pf[c][qt] = v;
      }
    }
    // O^T[dh][q] += V^T[dh][keys] P^T[keys][q]; A slots follow the same key permutation
#pragma unroll
    for (int d = 0; d < 4; ++d) {
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const bf16* vrow = &Vs[buf][d * 16 + lr][c * 32 + g * 4];
        const bf16x4 lo = *reinterpret_cast<const bf16x4*>(vrow);
        const bf16x4 hi = *reinterpret_cast<const bf16x4*>(vrow + 16);
        const bf16x8 vf = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
#pragma unroll
        for (int qt = 0; qt < QT; ++qt)
          o[d][qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[c][qt], o[d][qt], 0, 0, 0);
      }
    }
  };

  const int nkb = a.Tpad / kKB;
  static_for<PF>([&](auto P) __attribute__((always_inline)) {
    if (decltype(P)::value < nkb) gload(P, decltype(P)::value * kKB);
  });
  sstore(std::integral_constant<int, 0>{}, 0);
  __syncthreads();
  // Full groups of PF tiles run branch-free (prefetch index clamped to the
  // last tile; a store after the last tile goes to a buffer nobody reads
  // again) so that PF tiles stay in flight.  The last tile is kept out of the
  // groups: it runs last, with the key mask.
  const std::integral_constant<bool, false> nomask{};
  const std::integral_constant<bool, true> withmask{};
  const int nbody = nkb - 1;
  const int nfull = nbody / PF * PF;
  for (int kb0 = 0; kb0 < nfull; kb0 += PF) {
    static_for<PF>([&](auto J) __attribute__((always_inline)) {
      constexpr int j = decltype(J)::value;
      const int kb = kb0 + j;
      gload(J, min(kb + PF, nkb - 1) * kKB);  // slot j held tile kb, already in LDS
      block(kb & 1, kb * kKB, nomask);
      sstore(std::integral_constant<int, (j + 1) % PF>{}, (kb + 1) & 1);
      __syncthreads();
    });
  }
  static_for<PF>([&](auto J) __attribute__((always_inline)) {
    constexpr int j = decltype(J)::value;
    const int kb = nfull + j;
    if (kb < nbody) {
      block(kb & 1, kb * kKB, nomask);
      sstore(std::integral_constant<int, (j + 1) % PF>{}, (kb + 1) & 1);
      __syncthreads();
    }
  });
  block(nbody & 1, nbody * kKB, withmask);

  // normalise and store O[b*T + q][h*64 + dh]; lane holds dh = d*16 + 4g + r of query lr
  bf16* out = static_cast<bf16*>(a.out);
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    float l = lrun[qt];
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    const float inv = 1.0f / l;
    const int q = q0 + qt * 16 + lr;
    if (q >= a.T) continue;
    bf16* orow = out + ((size_t)b * a.T + q) * a.D + h * kDh;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      bf16x4 v;
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = static_cast<bf16>(o[d][qt][r] * inv);
      *reinterpret_cast<bf16x4*>(orow + d * 16 + g * 4) = v;
    }
  }
}

// ------------------------------------------------------------- fp32 attention
// One thread per query, online softmax over all keys (parity mode only).
template <int DH>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgs a) {
  if (a.skip && *a.skip) return;
  const int bh = blockIdx.y;
  const int b = bh / a.H, h = bh % a.H;
  const int q = blockIdx.x * 64 + threadIdx.x;
  if (q >= a.T) return;
  const float* Q = static_cast<const float*>(a.q) + ((size_t)bh * a.Tpad + q) * DH;
  const float* Kg = static_cast<const float*>(a.k) + (size_t)bh * a.Tpad * DH;
  const float* Vt = static_cast<const float*>(a.vt) + (size_t)bh * DH * a.Tpad;
  float qv[DH], acc[DH];
  const float sc = rsqrtf((float)DH);
#pragma unroll
  for (int d = 0; d < DH; ++d) {
    qv[d] = Q[d] * sc;
    acc[d] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int j = 0; j < a.T; ++j) {
    float s = 0.f;
#pragma unroll
    for (int d = 0; d < DH; ++d) s += qv[d] * Kg[(size_t)j * DH + d];
    const float mn = fmaxf(m, s);
    const float corr = __expf(m - mn);
    const float p = __expf(s - mn);
    l = l * corr + p;
#pragma unroll
    for (int d = 0; d < DH; ++d) acc[d] = acc[d] * corr + p * Vt[(size_t)d * a.Tpad + j];
    m = mn;
  }
  float* orow = static_cast<float*>(a.out) + ((size_t)b * a.T + q) * a.D + h * DH;
  const float inv = 1.0f / l;
#pragma unroll
  for (int d = 0; d < DH; ++d) orow[d] = acc[d] * inv;
}

}  // namespace

hipError_t launch_qkv_relayout(const RelayoutArgs& a, bool bf16_mode, hipStream_t s) {
  dim3 grid((a.T + 63) / 64, a.H, a.B);
  if (a.dh == 64) {
    if (bf16_mode) launch_k(qkv_relayout_kernel<bf16, 64>, grid, 256, 0, s, a);
    else launch_k(qkv_relayout_kernel<float, 64>, grid, 256, 0, s, a);
  } else if (a.dh == 32) {
    if (bf16_mode) launch_k(qkv_relayout_kernel<bf16, 32>, grid, 256, 0, s, a);
    else launch_k(qkv_relayout_kernel<float, 32>, grid, 256, 0, s, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// grid for qt query tiles per wave and nw waves per block
// (qt, nw, pf): query tiles of 16 per wave, waves per block, K/V tiles in
// flight.  Only the instantiated combinations are accepted.
hipError_t launch_attention_cfg(const AttnArgs& a, int qt, int nw, int pf, hipStream_t s) {
  if (a.dh != kDh || a.Tpad % kKB) return hipErrorInvalidValue;
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)a.dh);
  const int qb = qt * nw * 16;
  const dim3 grid((a.T + qb - 1) / qb, a.B * a.H);
  const int key = qt * 10000 + nw * 100 + pf;
  switch (key) {
    case 10203: launch_k(attn_bf16_kernel<1, 2, 3>, grid, 128, 0, s, a, scale_log2); break;
    case 10207: launch_k(attn_bf16_kernel<1, 2, 7>, grid, 128, 0, s, a, scale_log2); break;
    case 10403: launch_k(attn_bf16_kernel<1, 4, 3>, grid, 256, 0, s, a, scale_log2); break;
    case 10407: launch_k(attn_bf16_kernel<1, 4, 7>, grid, 256, 0, s, a, scale_log2); break;
    case 10803: launch_k(attn_bf16_kernel<1, 8, 3>, grid, 512, 0, s, a, scale_log2); break;
    case 20403: launch_k(attn_bf16_kernel<2, 4, 3>, grid, 256, 0, s, a, scale_log2); break;
    case 20803: launch_k(attn_bf16_kernel<2, 8, 3>, grid, 512, 0, s, a, scale_log2); break;
    case 20805: launch_k(attn_bf16_kernel<2, 8, 5>, grid, 512, 0, s, a, scale_log2); break;
    case 40402: launch_k(attn_bf16_kernel<4, 4, 2>, grid, 256, 0, s, a, scale_log2); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attention(const AttnArgs& a, bool bf16_mode, hipStream_t s) {
  if (bf16_mode) {
    // 8 waves x 32 queries with 5 K/V tiles in flight when that still fills
    // the chip, else 4 waves x 16 queries
    const long blocks = (long)((a.T + 255) / 256) * a.B * a.H;
    if (blocks >= 256) return launch_attention_cfg(a, 2, 8, 5, s);
    return launch_attention_cfg(a, 1, 4, 3, s);
  }
  dim3 grid((a.T + 63) / 64, a.B * a.H);
  if (a.dh == 64) launch_k(attn_f32_kernel<64>, grid, 64, 0, s, a);
  else if (a.dh == 32) launch_k(attn_f32_kernel<32>, grid, 64, 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace wam
