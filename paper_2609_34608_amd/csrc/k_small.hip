// Bandwidth- and latency-bound kernels of the denoising step and of the
// state-adaptation operators (gfx950, wave64).
#include <math.h>

#include <algorithm>
#include <mutex>
#include <string>

#include "wam_internal.h"

namespace wam {

namespace {

constexpr int kMaxVpl = 32;  // row kernels hold D/64 <= 32 values per lane

__device__ __forceinline__ double block_sum_d(double v, double* sh) {
  v = wave_sum_d(v);
  const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int nw = blockDim.x / kWave;
  __syncthreads();
  if (lane == 0) sh[w] = v;
  __syncthreads();
  double t = 0.0;
  for (int i = 0; i < nw; ++i) t += sh[i];
  return t;
}

// ------------------------------------------------------------- timestep MLP
// Small GEMV for the conditioning MLP: block = 64 outputs x 16 K-groups,
// y[n] = SiLU(sum_k x[k] W[k][n] + b[n]).  With FEATURES the input is
// computed in-kernel from sigma: x = [cos(t f_i), sin(t f_i)], t = 1000 sigma,
// f_i = 10000^(-i/128) (float64 arguments).
constexpr int kTimeDim = 256;
constexpr int kSgN = 64, kSgK = 16;
template <bool FEATURES>
__global__ __launch_bounds__(kSgN* kSgK) void small_gemv_silu_kernel(float sigma, const float* __restrict__ x,
                                                                    const float* __restrict__ W,
                                                                    const float* __restrict__ b,
                                                                    float* __restrict__ y, int K, int N) {
  __shared__ float xs[2048];
  __shared__ float part[kSgK][kSgN + 1];
  const int tid = threadIdx.x, nl = tid % kSgN, kg = tid / kSgN;
  for (int k = tid; k < K; k += blockDim.x) {
    if constexpr (FEATURES) {
      const int half = K / 2;
      const int j = k < half ? k : k - half;
      const double t = 1000.0 * (double)sigma;
      const double f = exp(-log(10000.0) * (double)j / (double)half);
      xs[k] = (float)(k < half ? cos(t * f) : sin(t * f));
    } else {
      xs[k] = x[k];
    }
  }
  __syncthreads();
  const int n = blockIdx.x * kSgN + nl;
  float acc = 0.f;
  if (n < N) {
#pragma unroll 4
    for (int k = kg; k < K; k += kSgK) acc += xs[k] * W[(size_t)k * N + n];
  }
  part[kg][nl] = acc;
  __syncthreads();
  if (kg == 0 && n < N) {
    float s = b[n];
    for (int g = 0; g < kSgK; ++g) s += part[g][nl];
    y[n] = s / (1.0f + __expf(-s));
  }
}

// ------------------------------------------------------------- GEMV
constexpr int kGemvKc = 32;   // input rows per split
constexpr int kGemvVec = 4;   // outputs per thread

__device__ __forceinline__ float act_apply(float v, int act) {
  return act == 1 ? v / (1.0f + __expf(-v)) : v;
}

template <typename TW>
__global__ void gemv_partial_kernel(const float* __restrict__ x, const TW* __restrict__ W,
                                    float* __restrict__ partial, int K, int N, int in_act) {
  const int n0 = (blockIdx.x * blockDim.x + threadIdx.x) * kGemvVec;
  const int k0 = blockIdx.y * kGemvKc;
  if (n0 >= N) return;
  float acc[kGemvVec] = {0.f, 0.f, 0.f, 0.f};
  const int k1 = min(K, k0 + kGemvKc);
  for (int k = k0; k < k1; ++k) {
    const float xv = act_apply(x[k], in_act);
    const TW* row = W + (size_t)k * N + n0;
#pragma unroll
    for (int j = 0; j < kGemvVec; ++j) acc[j] += xv * to_f32(row[j]);
  }
  float* p = partial + (size_t)blockIdx.y * N + n0;
#pragma unroll
  for (int j = 0; j < kGemvVec; ++j) p[j] = acc[j];
}

__global__ void gemv_reduce_kernel(const float* __restrict__ partial, const float* __restrict__ b,
                                   float* __restrict__ y, int nchunk, int N, int out_act) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= N) return;
  float s = 0.f;
  for (int c = 0; c < nchunk; ++c) s += partial[(size_t)c * N + n];
  y[n] = act_apply(s + b[n], out_act);
}

// ------------------------------------------------------------- embedding
// h[b,t,:] = token (video | action | obs) @ W_branch + b_branch + PE(t), PE a
// table built once at init
__global__ void embed_kernel(EmbedArgs a) {
  const int row = blockIdx.x;  // b*T + t
  const int b = row / a.T, t = row % a.T;
  __shared__ float tok[64];
  const float* w;
  const float* bias;
  int c;
  const int traj = a.Nv * a.Cv + a.Na * a.A;
  if (t < a.Nv) {
    c = a.Cv;
    w = a.wv;
    bias = a.bv;
    if (threadIdx.x < c) tok[threadIdx.x] = a.x[(size_t)b * traj + (size_t)t * a.Cv + threadIdx.x];
  } else if (t < a.Nv + a.Na) {
    c = a.A;
    w = a.wa;
    bias = a.ba;
    if (threadIdx.x < c)
      tok[threadIdx.x] = a.x[(size_t)b * traj + (size_t)a.Nv * a.Cv + (size_t)(t - a.Nv) * a.A + threadIdx.x];
  } else {
    c = a.Co;
    w = a.wo;
    bias = a.bo;
    if (threadIdx.x < c)
      tok[threadIdx.x] = a.cond[((size_t)b * a.No + (t - a.Nv - a.Na)) * a.Co + threadIdx.x];
  }
  __syncthreads();
  const float* pe = a.pe + (size_t)t * a.D;
  for (int d = threadIdx.x; d < a.D; d += blockDim.x) {
    float s = bias[d];
    for (int j = 0; j < c; ++j) s += tok[j] * w[(size_t)j * a.D + d];
    a.h[(size_t)row * a.D + d] = s + pe[d];
  }
}

// Vectorised form: a block takes up to R consecutive rows of one branch
// (video, action or observation tokens) of one sample, so that the branch's
// weight rows are read once for all of them (with one row per block the
// weight reads from L2 outweighed the HBM traffic of long sequences: 66 ->
// 33 us at T = 10176 with R = 8); thread i owns columns 4i..4i+3 (D / 4
// threads).  Every load a thread needs (bias, the up to kEmbedC weight rows,
// clamped to the branch's channel count against zero-padded token values,
// and the position-embedding rows) is issued before the sums.
constexpr int kEmbedC = 16;
__host__ __device__ inline int embed_blocks_per_sample(int Nv, int Na, int No, int R) {
  return (Nv + R - 1) / R + (Na + R - 1) / R + (No + R - 1) / R;
}
template <int R>
__global__ __launch_bounds__(512) void embed_v4_kernel(EmbedArgs a) {
  constexpr int kEmbedRows = R;
  const int per = embed_blocks_per_sample(a.Nv, a.Na, a.No, R);
  const int b = blockIdx.x / per, j = blockIdx.x % per;
  const int gv = (a.Nv + kEmbedRows - 1) / kEmbedRows, ga = (a.Na + kEmbedRows - 1) / kEmbedRows;
  const float* w;
  const float* bias;
  const float* src;  // token values of the block's first row
  int c, t0, n;      // channels, first row (within the sample), rows of this block
  const int traj = a.Nv * a.Cv + a.Na * a.A;
  if (j < gv) {
    t0 = j * kEmbedRows, n = min(kEmbedRows, a.Nv - t0), c = a.Cv, w = a.wv, bias = a.bv;
    src = a.x + (size_t)b * traj + (size_t)t0 * a.Cv;
  } else if (j < gv + ga) {
    const int i0 = (j - gv) * kEmbedRows;
    t0 = a.Nv + i0, n = min(kEmbedRows, a.Na - i0), c = a.A, w = a.wa, bias = a.ba;
    src = a.x + (size_t)b * traj + (size_t)a.Nv * a.Cv + (size_t)i0 * a.A;
  } else {
    const int i0 = (j - gv - ga) * kEmbedRows;
    t0 = a.Nv + a.Na + i0, n = min(kEmbedRows, a.No - i0), c = a.Co, w = a.wo, bias = a.bo;
    src = a.cond + ((size_t)b * a.No + i0) * a.Co;
  }
  __shared__ float tok[kEmbedRows][kEmbedC];
  for (int i = threadIdx.x; i < kEmbedRows * kEmbedC; i += blockDim.x) {
    const int r = i / kEmbedC, ch = i % kEmbedC;
    tok[r][ch] = r < n && ch < c ? src[(size_t)r * c + ch] : 0.f;
  }
  const int col = threadIdx.x * 4;
  const bool live = col < a.D;
  const int cc = live ? col : 0;
  const f32x4 b4 = *reinterpret_cast<const f32x4*>(bias + cc);
  f32x4 w4[kEmbedC], p4[kEmbedRows];
#pragma unroll
  for (int k = 0; k < kEmbedC; ++k) w4[k] = *reinterpret_cast<const f32x4*>(w + (size_t)min(k, c - 1) * a.D + cc);
#pragma unroll
  for (int r = 0; r < kEmbedRows; ++r)
    p4[r] = *reinterpret_cast<const f32x4*>(a.pe + (size_t)(t0 + min(r, n - 1)) * a.D + cc);
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kEmbedRows; ++r) {
    if (r >= n) break;
    f32x4 acc = b4;
#pragma unroll
    for (int k = 0; k < kEmbedC; ++k) acc += tok[r][k] * w4[k];
    if (live) *reinterpret_cast<f32x4*>(a.h + ((size_t)b * a.T + t0 + r) * a.D + col) = acc + p4[r];
  }
}

// ------------------------------------------------------------- LN + modulation
// One wave per row; lane holds elements lane + 64 i.
template <typename TOut>
__global__ void ln_modulate_kernel(const float* __restrict__ h, const float* __restrict__ shift,
                                   const float* __restrict__ scale, TOut* __restrict__ u,
                                   int rows, int D, float eps, const int* skip) {
  if (skip && *skip) return;
  const int row = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  if (row >= rows) return;
  const float* hr = h + (size_t)row * D;
  const int vpl = D / kWave;
  float v[kMaxVpl];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kMaxVpl; ++i) {
    if (i < vpl) {
      v[i] = hr[lane + kWave * i];
      s += v[i];
    }
  }
  const float mean = wave_sum(s) / (float)D;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < kMaxVpl; ++i)
    if (i < vpl) {
      const float d = v[i] - mean;
      q += d * d;
    }
  const float rstd = rsqrtf(wave_sum(q) / (float)D + eps);
  TOut* ur = u + (size_t)row * D;
#pragma unroll
  for (int i = 0; i < kMaxVpl; ++i)
    if (i < vpl) {
      const int c = lane + kWave * i;
      ur[c] = from_f32<TOut>((v[i] - mean) * rstd * (1.0f + scale[c]) + shift[c]);
    }
}

// Vectorised form for D % 256 == 0 and bf16 output: lane holds
// elements 4 lane + 256 i .. +3 (16-byte loads, 8-byte stores).  N4 = D / 256
// is a template argument so that the row and the modulation are fetched by
// 3 N4 loads issued together, ahead of the reductions (with a run-time count
// the compiler emitted one load and one wait per chunk).
template <int N4>
__global__ __launch_bounds__(256) void ln_modulate_v4_kernel(const float* __restrict__ h, const float* __restrict__ shift,
                                                             const float* __restrict__ scale, bf16* __restrict__ u,
                                                             int rows, float eps, const int* skip) {
  if (skip && *skip) return;
  constexpr int D = N4 * 256;
  const int row = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  if (row >= rows) return;
  const f32x4* hr = reinterpret_cast<const f32x4*>(h + (size_t)row * D);
  const f32x4* sc4 = reinterpret_cast<const f32x4*>(scale);
  const f32x4* sh4 = reinterpret_cast<const f32x4*>(shift);
  f32x4 v[N4], sc[N4], sh[N4];
#pragma unroll
  for (int i = 0; i < N4; ++i) v[i] = hr[lane + kWave * i];
#pragma unroll
  for (int i = 0; i < N4; ++i) {
    sc[i] = sc4[lane + kWave * i];
    sh[i] = sh4[lane + kWave * i];
  }
  __builtin_amdgcn_sched_barrier(0);  // keep the modulation loads ahead of the reductions
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < N4; ++i) s += (v[i].x + v[i].y) + (v[i].z + v[i].w);
  const float mean = wave_sum(s) / (float)D;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < N4; ++i) {
    const float a = v[i].x - mean, b = v[i].y - mean, c = v[i].z - mean, d = v[i].w - mean;
    q += (a * a + b * b) + (c * c + d * d);
  }
  const float rstd = rsqrtf(wave_sum(q) / (float)D + eps);
#pragma unroll
  for (int i = 0; i < N4; ++i) {
    const int c = 4 * (lane + kWave * i);
    bf16x4 o = {static_cast<bf16>((v[i].x - mean) * rstd * (1.0f + sc[i].x) + sh[i].x),
                static_cast<bf16>((v[i].y - mean) * rstd * (1.0f + sc[i].y) + sh[i].y),
                static_cast<bf16>((v[i].z - mean) * rstd * (1.0f + sc[i].z) + sh[i].z),
                static_cast<bf16>((v[i].w - mean) * rstd * (1.0f + sc[i].w) + sh[i].w)};
    *reinterpret_cast<bf16x4*>(u + (size_t)row * D + c) = o;
  }
}

// ------------------------------------------------------------- final layer + Euler
// A block of NW waves takes NW R consecutive trajectory rows of one branch of
// one sample, wave w the rows w R .. w R + R-1, so that all of them share the
// branch's head weights (W^T packed [Cout][D]) and the modulation vectors,
// which the block copies from global memory into LDS once.  A lane holds elements VEC lane + 64 VEC i ..
// + VEC-1 of each row.  Every load that does not depend on a reduction is
// issued up front (the rows, the modulation, the weight copy).  Each lane
// forms partial products of its elements for R rows x 16 channels; butterfly
// sums over the 64 lanes leave lane l < 16 R with the full dot product of row
// l / 16, channel l % 16, which it stores as the velocity and/or applies as
// the Euler update x += dsigma v.
constexpr int kFinalCout = 16;
template <int VEC>
using fvec = float __attribute__((ext_vector_type(VEC)));

// Copies n floats (a multiple of 4) from global memory to LDS with
// direct-to-LDS 16-byte loads, 1 KiB per instruction, runs c = first, first +
// step, ...: lanes past the end of the last run re-read the final 16 bytes,
// into LDS that is never read (the destination is sized in whole runs).
__device__ __forceinline__ void copy_to_lds(const float* src, float* dst, int n, int lane, int first, int step) {
  for (int c = first; c * 256 < n; c += step) {
    const int e = c * 256 + 4 * lane;
    __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(src + (e < n ? e : n - 4)),
                                     (__attribute__((address_space(3))) void*)(dst + c * 256), 16, 0, 0);
  }
}

// D a multiple of 64 VEC, at most 64 VEC MAXC.  Each wave first requests its
// rows (HBM; rows at or past the branch end re-read the group's first row and
// are never stored), then the block copies the Cout x D weights (contiguous,
// the same layout in LDS) and the modulation vectors into LDS; after a full
// wait and the barrier each wave reads its columns of them from LDS.
template <int VEC, int R, int MAXC, int NW>
__global__ __launch_bounds__(NW * 64) void final_kernel(FinalArgs a) {
  using vec = fvec<VEC>;
  constexpr int DMAX = MAXC * 64 * VEC;  // a multiple of 256
  __shared__ __attribute__((aligned(1024))) float wsm[kFinalCout * DMAX];
  __shared__ __attribute__((aligned(1024))) float msc[DMAX], msh[DMAX];
  const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
  constexpr int RB = NW * R;  // rows per block
  const int gv = (a.Nv + RB - 1) / RB, ga = (a.Na + RB - 1) / RB, per = gv + ga;
  const int b = blockIdx.x / per, j = blockIdx.x % per;
  const bool video = j < gv;
  const int t0 = (video ? j * RB : a.Nv + (j - gv) * RB) + wid * R;
  const int tend = video ? a.Nv : a.Nv + a.Na;
  const bool active = t0 < tend;  // waves past the branch end only help with the copies
  const int nch = a.D / (kWave * VEC);
  auto col = [&](int i) { return VEC * lane + kWave * VEC * i; };
  vec u[R][MAXC];
  if (active) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const float* hr = a.h + ((size_t)b * a.T + (t0 + r < tend ? t0 + r : t0)) * a.D;
#pragma unroll
      for (int i = 0; i < MAXC; ++i)
        if (i < nch) u[r][i] = *reinterpret_cast<const vec*>(hr + col(i));
    }
  }
  const int cout = video ? a.Cv : a.A;
  copy_to_lds(video ? a.wv : a.wa, wsm, cout * a.D, lane, wid, NW);
  copy_to_lds(a.scale, msc, a.D, lane, (wid + NW - 1) % NW, NW);
  copy_to_lds(a.shift, msh, a.D, lane, (wid + NW - 2) % NW, NW);
  // the compiler does not track the LDS writes of those loads: wait for all
  // of this wave's memory operations, then for every wave's
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (!active) return;

  float mean[R], rstd[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < MAXC; ++i)
      if (i < nch)
#pragma unroll
        for (int e = 0; e < VEC; ++e) s += u[r][i][e];
    mean[r] = wave_sum(s) / (float)a.D;
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    float q = 0.f;
#pragma unroll
    for (int i = 0; i < MAXC; ++i)
      if (i < nch)
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const float dv = u[r][i][e] - mean[r];
          q += dv * dv;
        }
    rstd[r] = rsqrtf(wave_sum(q) / (float)a.D + a.eps);
  }
#pragma unroll
  for (int i = 0; i < MAXC; ++i)
    if (i < nch) {
      const vec sc = *reinterpret_cast<const vec*>(msc + col(i));
      const vec sh = *reinterpret_cast<const vec*>(msh + col(i));
#pragma unroll
      for (int r = 0; r < R; ++r) u[r][i] = (u[r][i] - mean[r]) * rstd[r] * (1.0f + sc) + sh;
    }
  constexpr int NV = R * kFinalCout;  // partial sums per lane, index r * 16 + o
  float v[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k) v[k] = 0.f;
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    if (i < nch) {
      vec w[kFinalCout];
#pragma unroll
      for (int o = 0; o < kFinalCout; ++o)
        w[o] = o < cout ? *reinterpret_cast<const vec*>(wsm + o * a.D + col(i)) : vec(0.f);
#pragma unroll
      for (int r = 0; r < R; ++r)
#pragma unroll
        for (int o = 0; o < kFinalCout; ++o) {
          const vec p = u[r][i] * w[o];
#pragma unroll
          for (int e = 0; e < VEC; ++e) v[r * kFinalCout + o] += p[e];
        }
    }
  }
  // lane bits above NV: plain butterfly sums; then a reduce-scatter, where
  // after the step over lane bit s, v[k] (k < s) holds the partial sum of
  // index k + (lane & s) + the bits already consumed.  Lane l ends with the
  // full sum of index l % NV.
#pragma unroll
  for (int s = kWave / 2; s >= NV; s >>= 1)
#pragma unroll
    for (int k = 0; k < NV; ++k) v[k] += __shfl_xor(v[k], s, 64);
#pragma unroll
  for (int s = NV / 2; s >= 1; s >>= 1) {
    const bool hi = (lane & s) != 0;
#pragma unroll
    for (int k = 0; k < s; ++k) {
      const float keep = hi ? v[k + s] : v[k];
      const float send = hi ? v[k] : v[k + s];
      v[k] = keep + __shfl_xor(send, s, 64);
    }
  }
  const int r = lane / kFinalCout, o = lane % kFinalCout, t = t0 + r;
  if (lane >= NV || t >= tend || o >= cout) return;
  const float vel = v[0] + (video ? a.bv : a.ba)[o];
  const int traj = a.Nv * a.Cv + a.Na * a.A;
  const size_t idx = (size_t)b * traj + (video ? (size_t)t * a.Cv + o
                                               : (size_t)a.Nv * a.Cv + (size_t)(t - a.Nv) * a.A + o);
  if (a.v_out) a.v_out[idx] = vel;
  if (a.x) a.x[idx] += a.dsigma * vel;
}


// ------------------------------------------------------------- Residual Rescaling
// Per row: sums of p_i p_a, p_i^2, p_a^2 with p_i = h_s - h_q (float64), one
// wave per row (any D multiple of 4); rr_finish_kernel reduces them.
__global__ void rr_row_sums_kernel(const float* __restrict__ hs, const float* __restrict__ hq,
                                       const float* __restrict__ pa, double* __restrict__ out,
                                       int rows, int D) {
  const int row = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  if (row >= rows) return;
  const size_t off = (size_t)row * D;
  double sip = 0.0, sii = 0.0, saa = 0.0;
  for (int c = lane * 4; c < D; c += kWave * 4) {
    const float4 s4 = *reinterpret_cast<const float4*>(hs + off + c);
    const float4 q4 = *reinterpret_cast<const float4*>(hq + off + c);
    const float4 a4 = *reinterpret_cast<const float4*>(pa + off + c);
    const float pi[4] = {s4.x - q4.x, s4.y - q4.y, s4.z - q4.z, s4.w - q4.w};
    const float pv[4] = {a4.x, a4.y, a4.z, a4.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      sip += (double)pi[j] * pv[j];
      sii += (double)pi[j] * pi[j];
      saa += (double)pv[j] * pv[j];
    }
  }
  sip = wave_sum_d(sip);
  sii = wave_sum_d(sii);
  saa = wave_sum_d(saa);
  if (lane == 0) {
    out[(size_t)row * 3 + 0] = sip;
    out[(size_t)row * 3 + 1] = sii;
    out[(size_t)row * 3 + 2] = saa;
  }
}

// alpha (Eq. crr-alpha), cos and relative fit error (Eq. crr-gate) of one
// (sample, branch) from its float64 sums over nrows rows of D elements.
__device__ void rr_gate_stats(const RRGateArgs& a, int b, int br, int nrows, double sip, double sii, double saa) {
  const double n = (double)nrows * (double)a.D;
  const double den = fmax(saa / n, (double)a.eps);
  double alpha = (sip / n) / den;
  alpha = fmin(fmax(alpha, (double)a.alpha_min), (double)a.alpha_max);
  const bool ok_norm = sii > 0.0 && saa > 0.0;
  const double cosv = ok_norm ? sip / sqrt(sii * saa) : 0.0;
  const double r2 = fmax(sii - 2.0 * alpha * sip + alpha * alpha * saa, 0.0);
  const double fit = sii > 0.0 ? sqrt(r2) / sqrt(sii) : INFINITY;
  const bool pass = ok_norm && cosv >= (double)a.gamma_cos && fit <= (double)a.gamma_fit;
  double* r = a.result + ((size_t)b * 2 + br) * 8;
  r[0] = sip;
  r[1] = sii;
  r[2] = saa;
  r[3] = alpha;
  r[4] = cosv;
  r[5] = fit;
  r[6] = pass ? 1.0 : 0.0;
  r[7] = 0.0;
}

// The gate in two launches, both in fixed summation orders.  Partials: blocks
// are laid out per (sample, branch): sample b owns gV = ceil(nV / 4) blocks
// over the rows of branch 0 (rows [0, Nv) then [Nv+Na, T), nV = T - Na of
// them) followed by gA = ceil(Na / 4) over branch 1 (rows [Nv, Nv+Na)).  Wave
// w of a block takes one row (all of its loads issued before any
// arithmetic), and the block adds its rows in wave order into one partial
// (row_sums[block][3]).  The second kernel, one block per (sample, branch),
// adds that pair's partials in block order and writes the statistics.
template <int MAXV>
__global__ __launch_bounds__(256) void rr_gate_partials_kernel(RRGateArgs a) {
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  const int nV = a.T - a.Na;
  const int gV = (nV + 3) / 4, gA = (a.Na + 3) / 4, per = gV + gA;
  const int b = blockIdx.x / per, j = blockIdx.x % per;
  const bool br1 = j >= gV;
  const int i = (br1 ? j - gV : j) * 4 + w;  // row within the branch
  const bool valid = i < (br1 ? a.Na : nV);
  const int t = br1 ? a.Nv + i : (i < a.Nv ? i : i + a.Na);
  __shared__ double part[4][3];
  double sip = 0.0, sii = 0.0, saa = 0.0;
  if (valid) {
    const size_t off = ((size_t)b * a.T + t) * a.D;
    const int nv = a.D / (4 * kWave);
    const f32x4* s4 = reinterpret_cast<const f32x4*>(a.hs + off);
    const f32x4* q4 = reinterpret_cast<const f32x4*>(a.hq + off);
    const f32x4* a4 = reinterpret_cast<const f32x4*>(a.pa + off);
    f32x4 sv[MAXV], qv[MAXV], av[MAXV];
#pragma unroll
    for (int k = 0; k < MAXV; ++k)
      if (k < nv) {
        sv[k] = s4[lane + kWave * k];
        qv[k] = q4[lane + kWave * k];
        av[k] = a4[lane + kWave * k];
      }
#pragma unroll
    for (int k = 0; k < MAXV; ++k)
      if (k < nv) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const double pi = (double)(sv[k][e] - qv[k][e]), pv = (double)av[k][e];
          sip += pi * pv;
          sii += pi * pi;
          saa += pv * pv;
        }
      }
    sip = wave_sum_d(sip);
    sii = wave_sum_d(sii);
    saa = wave_sum_d(saa);
  }
  if (lane == 0) {
    part[w][0] = sip;
    part[w][1] = sii;
    part[w][2] = saa;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double* out = a.row_sums + (size_t)blockIdx.x * 3;
    out[0] = (part[0][0] + part[1][0]) + (part[2][0] + part[3][0]);
    out[1] = (part[0][1] + part[1][1]) + (part[2][1] + part[3][1]);
    out[2] = (part[0][2] + part[1][2]) + (part[2][2] + part[3][2]);
  }
}

__global__ __launch_bounds__(256) void rr_gate_finish_kernel(RRGateArgs a) {
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  const int b = blockIdx.x / 2, br = blockIdx.x % 2;
  const int nV = a.T - a.Na;
  const int gV = (nV + 3) / 4, gA = (a.Na + 3) / 4, per = gV + gA;
  const int first = b * per + (br ? gV : 0), cnt = br ? gA : gV;
  double s[3] = {0.0, 0.0, 0.0};
#pragma unroll 8
  for (int k = threadIdx.x; k < cnt; k += 256) {
    const double* p = a.row_sums + (size_t)(first + k) * 3;
    s[0] += p[0];
    s[1] += p[1];
    s[2] += p[2];
  }
  __shared__ double sh[3][4];
#pragma unroll
  for (int c = 0; c < 3; ++c) {
    const double v = wave_sum_d(s[c]);
    if (lane == 0) sh[c][w] = v;
  }
  __syncthreads();
  if (threadIdx.x == 0)
    rr_gate_stats(a, b, br, br ? a.Na : nV, (sh[0][0] + sh[0][1]) + (sh[0][2] + sh[0][3]),
                  (sh[1][0] + sh[1][1]) + (sh[1][2] + sh[1][3]), (sh[2][0] + sh[2][1]) + (sh[2][2] + sh[2][3]));
}

// One block per (sample, branch): alpha (Eq. crr-alpha), cos and relative
// fit error (Eq. crr-gate) from the float64 row sums.
__global__ __launch_bounds__(1024) void rr_finish_kernel(RRGateArgs a) {
  const int b = blockIdx.x / 2, br = blockIdx.x % 2;
  __shared__ double sh[3][16];
  double s[3] = {0.0, 0.0, 0.0};
  // branch rows as one index range: A = [Nv, Nv+Na); V = [0, Nv) then [Nv+Na, T)
  const int nrows = br == 1 ? a.Na : a.T - a.Na;
  const double* base = a.row_sums + (size_t)b * a.T * 3;
#pragma unroll 4
  for (int i = threadIdx.x; i < nrows; i += blockDim.x) {
    const int t = br == 1 ? a.Nv + i : (i < a.Nv ? i : i + a.Na);
    s[0] += base[(size_t)t * 3 + 0];
    s[1] += base[(size_t)t * 3 + 1];
    s[2] += base[(size_t)t * 3 + 2];
  }
  const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  for (int j = 0; j < 3; ++j) {
    const double v = wave_sum_d(s[j]);
    if (lane == 0) sh[j][w] = v;
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  const int nw = blockDim.x / kWave;
  double sip = 0.0, sii = 0.0, saa = 0.0;
  for (int i = 0; i < nw; ++i) {
    sip += sh[0][i];
    sii += sh[1][i];
    saa += sh[2][i];
  }
  rr_gate_stats(a, b, br, nrows, sip, sii, saa);
}

// h_e = h_s + alpha_{b,branch} R_a (Eq. residual-injection), in place on h.
// A thread updates kInjV float4 spaced one block width apart (all loads
// first; in the model one per thread measured fastest).  A float4 never
// straddles rows (D % 4 == 0); its sample and branch come from comparisons
// against the float4 offsets of the sample and branch boundaries (host:
// rows * D / 4 < 2^31).
constexpr int kInjV = 1;
__global__ __launch_bounds__(256) void rr_inject_kernel(float* __restrict__ h, const float* __restrict__ Ra,
                                                        const double* __restrict__ result, int B, int T, int D,
                                                        int Nv, int Na, const int* flag) {
  if (flag && *flag != 1) return;
  const int d4 = D / 4, td4 = T * d4, n4 = B * td4, lo = Nv * d4, hi = (Nv + Na) * d4;
  const int base = blockIdx.x * (256 * kInjV) + threadIdx.x;
  f32x4* h4 = reinterpret_cast<f32x4*>(h);
  const f32x4* r4 = reinterpret_cast<const f32x4*>(Ra);
  f32x4 hv[kInjV], rv[kInjV];
#pragma unroll
  for (int u = 0; u < kInjV; ++u) {
    const int i4 = base + 256 * u;
    if (i4 < n4) {
      hv[u] = h4[i4];
      rv[u] = r4[i4];
    }
  }
#pragma unroll
  for (int u = 0; u < kInjV; ++u) {
    const int i4 = base + 256 * u;
    if (i4 < n4) {
      int b = 0, r = i4;
      while (r >= td4) {
        r -= td4;
        ++b;
      }
      const int br = (r >= lo && r < hi) ? 1 : 0;
      const float al = (float)result[((size_t)b * 2 + br) * 8 + 3];
      h4[i4] = hv[u] + al * rv[u];
    }
  }
}

__global__ void rr_pre_middle_kernel(const float* __restrict__ h, float* __restrict__ hq,
                                     float* __restrict__ pa, int64_t n4, const int* flag) {
  if (flag && *flag != 0) return;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  const float4 hv = reinterpret_cast<const float4*>(h)[i];
  const float4 qv = reinterpret_cast<const float4*>(hq)[i];
  reinterpret_cast<float4*>(pa)[i] = make_float4(hv.x - qv.x, hv.y - qv.y, hv.z - qv.z, hv.w - qv.w);
  reinterpret_cast<float4*>(hq)[i] = hv;
}

__global__ void rr_refresh_kernel(const float* __restrict__ h, const float* __restrict__ hq,
                                  float* __restrict__ Ra, int64_t n4, const int* flag) {
  if (flag && *flag != 0) return;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  const float4 hv = reinterpret_cast<const float4*>(h)[i];
  const float4 qv = reinterpret_cast<const float4*>(hq)[i];
  reinterpret_cast<float4*>(Ra)[i] = make_float4(hv.x - qv.x, hv.y - qv.y, hv.z - qv.z, hv.w - qv.w);
}

// Device-side reuse decision: AND of the pass bits over samples and branches
// (or forced), written as a flag that predicates the following launches.
__global__ void rr_decide_kernel(const double* __restrict__ result, int B, int nbranch, int force_accept, int* flag,
                                 double* hist_stats, int* hist_flag) {
  if (threadIdx.x != 0) return;
  int all = 1;
  for (int i = 0; i < B * 2; ++i) {
    const double* r = result + (size_t)i * 8;
    if (i % 2 < nbranch) all &= r[6] != 0.0;
    hist_stats[i * 3 + 0] = r[3];
    hist_stats[i * 3 + 1] = r[4];
    hist_stats[i * 3 + 2] = r[5];
  }
  const int accept = force_accept ? 1 : all;
  *flag = accept;
  *hist_flag = accept;
}

// Condition of the action model of an independent pair: observation tokens,
// then context tokens (e.g. the video model's latent), zero-padded to Co.
__global__ void pack_condition_kernel(const float* __restrict__ obs, int n_obs, int c_obs,
                                      const float* __restrict__ ctx, int n_ctx, int c_ctx, int64_t ctx_stride,
                                      float* __restrict__ cond, int B, int Co) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int nt = n_obs + n_ctx;
  if (i >= (int64_t)B * nt * Co) return;
  const int c = (int)(i % Co);
  const int t = (int)((i / Co) % nt);
  const int b = (int)(i / ((int64_t)Co * nt));
  float v = 0.f;
  if (t < n_obs) {
    if (c < c_obs) v = obs[((int64_t)b * n_obs + t) * c_obs + c];
  } else if (c < c_ctx) {
    v = ctx[(int64_t)b * ctx_stride + (int64_t)(t - n_obs) * c_ctx + c];
  }
  cond[i] = v;
}

__global__ void copy_f32_kernel(const float* __restrict__ src, float* __restrict__ dst, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = src[i];
}

// float4 copy, four per thread spaced one block width apart (n4 float4)
__global__ __launch_bounds__(256) void copy_f32x4_kernel(const f32x4* __restrict__ src, f32x4* __restrict__ dst,
                                                         int64_t n4) {
  const int64_t base = (int64_t)blockIdx.x * 1024 + threadIdx.x;
  f32x4 v[4];
#pragma unroll
  for (int u = 0; u < 4; ++u)
    if (base + 256 * u < n4) v[u] = src[base + 256 * u];
#pragma unroll
  for (int u = 0; u < 4; ++u)
    if (base + 256 * u < n4) dst[base + 256 * u] = v[u];
}

// ------------------------------------------------------------- Trajectory Remapping
// Four consecutive floats p[0 .. cnt) (zeros past cnt): one 16-byte load when
// VEC (the caller has checked the alignment and cnt == 4), else scalar loads.
template <bool VEC>
__device__ __forceinline__ f32x4 load_group(const float* p, int64_t cnt) {
  if constexpr (VEC) {
    return *reinterpret_cast<const f32x4*>(p);
  } else {
    f32x4 v = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (u < cnt) v[u] = p[u];
    return v;
  }
}

// Float64 sum of ((p - q) * scale)^2 over elements [4 g0, min(4 g1, n)) of a
// run, by the 256 threads of a block: thread t takes the 4-element groups
// t, t + 256, ... (four groups in flight per step), and each group's elements
// in order.  Both instantiations add in exactly this order, so the result
// does not depend on whether the 16-byte path was taken.
template <bool VEC>
__device__ __forceinline__ double run_sq_sum(const float* p, const float* q, double scale, int64_t g0,
                                             int64_t g1, int64_t n) {
  const int64_t full = n / 4 < g1 ? n / 4 : g1;  // groups with all four elements
  double s = 0.0;
  int64_t g = g0 + threadIdx.x;
  for (; g + 3 * 256 < full; g += 4 * 256) {
    f32x4 x[4], y[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      x[u] = load_group<VEC>(p + 4 * (g + u * 256), 4);
      y[u] = load_group<VEC>(q + 4 * (g + u * 256), 4);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double d = ((double)x[u][e] - (double)y[u][e]) * scale;
        s = fma(d, d, s);
      }
  }
  for (; g < g1; g += 256) {
    const int64_t cnt = n - 4 * g < 4 ? n - 4 * g : 4;
    const f32x4 x = load_group<VEC>(p + 4 * g, VEC ? 4 : cnt), y = load_group<VEC>(q + 4 * g, VEC ? 4 : cnt);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (e < cnt) {
        const double d = ((double)x[e] - (double)y[e]) * scale;
        s = fma(d, d, s);
      }
  }
  return s;
}

// rms of (x^r - x_bar)/sigma_r per (sample, branch) over the whole branch, in
// two launches: each branch is cut into reduce_chunks(n) runs of whole
// 4-element groups, one block per run sums its squares (float64); then one
// block per (sample, branch) adds the run sums in a fixed order (the same
// bits on every call) and turns the rms into the remap coefficient
// sigma_b0 / (sigma_r rms) (0 for a zero direction).
template <bool VEC>
__global__ __launch_bounds__(256) void remap_partial_kernel(RemapArgs a) {
  __shared__ double sh[16];
  const int sb = blockIdx.y;  // sample * 2 + branch
  const int b = sb / 2, br = sb % 2;
  const int64_t traj = (int64_t)a.Nv * a.Cv + (int64_t)a.Na * a.A;
  const int64_t lo = br == 0 ? 0 : (int64_t)a.Nv * a.Cv;
  const int64_t n = br == 0 ? (int64_t)a.Nv * a.Cv : (int64_t)a.Na * a.A;
  const int nch = reduce_chunks(n);
  if ((int)blockIdx.x >= nch) return;
  const int64_t ng = (n + 3) / 4, per = (ng + nch - 1) / nch;
  const int64_t g0 = (int64_t)blockIdx.x * per;
  const int64_t g1 = g0 + per < ng ? g0 + per : ng;
  const size_t off = (size_t)b * traj + lo;
  double s = run_sq_sum<VEC>(a.x_r + off, a.x_bar + off, 1.0 / (double)a.sigma_r, g0, g1, n);
  s = block_sum_d(s, sh);
  if (threadIdx.x == 0) a.partial[(size_t)sb * kRemapChunks + blockIdx.x] = s;
}

// Fixed-order sum of run sums p[0 .. n): thread t adds runs t, t + 256, ...
// in turn, then the 256 thread sums combine as block_sum_d does.
__device__ __forceinline__ double runs_sum(const double* p, int n, double* sh) {
  double s = 0.0;
  for (int c = threadIdx.x; c < n; c += 256) s += p[c];
  return block_sum_d(s, sh);
}

__global__ __launch_bounds__(256) void remap_finish_kernel(RemapArgs a) {
  __shared__ double sh[16];
  const int sb = blockIdx.x;
  const int br = sb % 2;
  const int64_t n = br == 0 ? (int64_t)a.Nv * a.Cv : (int64_t)a.Na * a.A;
  const double s = runs_sum(a.partial + (size_t)sb * kRemapChunks, reduce_chunks(n), sh);
  if (threadIdx.x == 0) {
    // x = x_bar + sigma_b0 d with d = ((x^r - x_bar) / sigma_r) / rms
    const double rms = n > 0 ? sqrt(s / (double)n) : 0.0;
    a.coef[sb] = rms > 0.0 ? (double)a.sigma_b0 / ((double)a.sigma_r * rms) : 0.0;
  }
}

// x[j] = x_bar[j+shift] + sigma_b0 d[j+shift] on mapped slots, sigma_b0 eps[j]
// elsewhere.  Slot j of a branch of width w is mapped when j + shift < slots,
// i.e. when the element index within the branch plus shift * w stays inside
// the branch.  Grid (element groups, sample): with VEC each thread takes four
// consecutive elements with 16-byte loads and stores (the host has checked
// that the pointers, both branch lengths and both shifted offsets are
// multiples of four floats, so a group lies in one branch and is mapped or
// unmapped as a whole); otherwise one element per thread.  Every element is
// computed by the same expression either way.
__device__ __forceinline__ float remap_value(float xb, float xr, double coef) {
  const double x = (double)xb;
  return (float)(x + ((double)xr - x) * coef);
}

template <bool VEC>
__global__ __launch_bounds__(256) void remap_apply_kernel(RemapArgs a) {
  const int64_t traj = (int64_t)a.Nv * a.Cv + (int64_t)a.Na * a.A;
  const int64_t nv = (int64_t)a.Nv * a.Cv;
  const int b = blockIdx.y;
  const size_t base = (size_t)b * traj;
  if constexpr (VEC) {
    const int64_t i = 4 * ((int64_t)blockIdx.x * 256 + threadIdx.x);
    if (i >= traj) return;
    const bool video = i < nv;
    const int64_t src = i + (video ? (int64_t)a.shift_video * a.Cv : (int64_t)a.shift_action * a.A);
    f32x4 out;
    if (src < (video ? nv : traj)) {
      const f32x4 xb = *reinterpret_cast<const f32x4*>(a.x_bar + base + src);
      const f32x4 xr = *reinterpret_cast<const f32x4*>(a.x_r + base + src);
      const double c = a.coef[b * 2 + (video ? 0 : 1)];
#pragma unroll
      for (int e = 0; e < 4; ++e) out[e] = remap_value(xb[e], xr[e], c);
    } else {
      out = a.sigma_b0 * *reinterpret_cast<const f32x4*>(a.noise + base + i);
    }
    *reinterpret_cast<f32x4*>(a.x_out + base + i) = out;
  } else {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= traj) return;
    const bool video = i < nv;
    const int64_t src = i + (video ? (int64_t)a.shift_video * a.Cv : (int64_t)a.shift_action * a.A);
    a.x_out[base + i] = src < (video ? nv : traj)
                            ? remap_value(a.x_bar[base + src], a.x_r[base + src], a.coef[b * 2 + (video ? 0 : 1)])
                            : a.sigma_b0 * a.noise[base + i];
  }
}

// ------------------------------------------------------------- Observation Rebinding
struct OrSumArgs {
  const float* u_hat[WAM_MAX_COMPONENTS];
  const float* u[WAM_MAX_COMPONENTS];
  int64_t n[WAM_MAX_COMPONENTS];
  double inv_delta[WAM_MAX_COMPONENTS];
  double* sums;
};

// Run sums of ((u_hat - u) / delta)^2 of component blockIdx.y, run blockIdx.x
// of reduce_chunks(n) runs of whole 4-element groups (float64, the order of
// run_sq_sum); the host adds the runs in order.
template <bool VEC>
__global__ __launch_bounds__(256) void or_sums_kernel(OrSumArgs a) {
  __shared__ double sh[16];
  const int m = blockIdx.y;
  const int64_t n = a.n[m];
  const int nch = reduce_chunks(n);
  if ((int)blockIdx.x >= nch) return;
  const int64_t ng = (n + 3) / 4, per = (ng + nch - 1) / nch;
  const int64_t g0 = (int64_t)blockIdx.x * per;
  const int64_t g1 = g0 + per < ng ? g0 + per : ng;
  double s = run_sq_sum<VEC>(a.u_hat[m], a.u[m], a.inv_delta[m], g0, g1, n);
  s = block_sum_d(s, sh);
  if (threadIdx.x == 0) a.sums[(size_t)m * kRemapChunks + blockIdx.x] = s;
}

}  // namespace

// ================================================================ launchers
hipError_t launch_timestep_mlp(float sigma, const float* w1, const float* b1, const float* w2, const float* b2,
                               float* a1, float* silu_c, int D, hipStream_t s) {
  if (D > 2048) return hipErrorInvalidValue;
  const int grid = (D + kSgN - 1) / kSgN;
  launch_k(small_gemv_silu_kernel<true>, grid, kSgN * kSgK, 0, s, sigma, nullptr, w1, b1, a1, kTimeDim, D);
  launch_k(small_gemv_silu_kernel<false>, grid, kSgN * kSgK, 0, s, 0.f, a1, w2, b2, silu_c, D, D);
  return hipGetLastError();
}

hipError_t launch_gemv(const float* x, const void* W, bool w_bf16, const float* b, float* y,
                       float* partial, int K, int N, int in_act, int out_act, hipStream_t s) {
  if (N % kGemvVec) return hipErrorInvalidValue;
  const int nchunk = (K + kGemvKc - 1) / kGemvKc;
  dim3 grid((N / kGemvVec + 255) / 256, nchunk);
  if (w_bf16)
    launch_k(gemv_partial_kernel<bf16>, grid, 256, 0, s, x, (const bf16*)W, partial, K, N, in_act);
  else
    launch_k(gemv_partial_kernel<float>, grid, 256, 0, s, x, (const float*)W, partial, K, N, in_act);
  launch_k(gemv_reduce_kernel, (N + 255) / 256, 256, 0, s, partial, b, y, nchunk, N, out_act);
  return hipGetLastError();
}

hipError_t launch_embed(const EmbedArgs& a, hipStream_t s) {
  if (a.Cv > 64 || a.A > 64 || a.Co > 64) return hipErrorInvalidValue;
  // every branch present has at least one channel (the clamp reads row c-1)
  const bool chans = (a.Nv == 0 || a.Cv >= 1) && (a.Na == 0 || a.A >= 1) && (a.No == 0 || a.Co >= 1);
  if (a.D % 4 == 0 && a.D <= 2048 && a.Cv <= kEmbedC && a.A <= kEmbedC && a.Co <= kEmbedC && chans) {
    const int threads = (a.D / 4 + kWave - 1) / kWave * kWave;
    // rows per block: share the weight reads where the grid stays above
    // ~1000 blocks, one row per block for short sequences (latency)
    const long rows = (long)a.B * a.T;
    if (rows >= 8192)
      launch_k(embed_v4_kernel<8>, a.B * embed_blocks_per_sample(a.Nv, a.Na, a.No, 8), threads, 0, s, a);
    else if (rows >= 4096)
      launch_k(embed_v4_kernel<4>, a.B * embed_blocks_per_sample(a.Nv, a.Na, a.No, 4), threads, 0, s, a);
    else if (rows >= 2048)
      launch_k(embed_v4_kernel<2>, a.B * embed_blocks_per_sample(a.Nv, a.Na, a.No, 2), threads, 0, s, a);
    else
      launch_k(embed_v4_kernel<1>, a.B * embed_blocks_per_sample(a.Nv, a.Na, a.No, 1), threads, 0, s, a);
  } else {
    launch_k(embed_kernel, a.B * a.T, 256, 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_ln_modulate(const float* h, const float* shift, const float* scale, void* u,
                              int rows, int D, float eps, bool bf16_out, hipStream_t s, const int* skip) {
  if (D % kWave || D / kWave > kMaxVpl) return hipErrorInvalidValue;
  const int wpb = 4;
  dim3 grid((rows + wpb - 1) / wpb);
  if (bf16_out && D % 256 == 0 && D <= 2048) {
    switch (D / 256) {
      case 1: launch_k(ln_modulate_v4_kernel<1>, grid, wpb * kWave, 0, s, h, shift, scale, (bf16*)u, rows, eps, skip); break;
      case 2: launch_k(ln_modulate_v4_kernel<2>, grid, wpb * kWave, 0, s, h, shift, scale, (bf16*)u, rows, eps, skip); break;
      case 3: launch_k(ln_modulate_v4_kernel<3>, grid, wpb * kWave, 0, s, h, shift, scale, (bf16*)u, rows, eps, skip); break;
      case 4: launch_k(ln_modulate_v4_kernel<4>, grid, wpb * kWave, 0, s, h, shift, scale, (bf16*)u, rows, eps, skip); break;
      case 5: launch_k(ln_modulate_v4_kernel<5>, grid, wpb * kWave, 0, s, h, shift, scale, (bf16*)u, rows, eps, skip); break;
      case 6: launch_k(ln_modulate_v4_kernel<6>, grid, wpb * kWave, 0, s, h, shift, scale, (bf16*)u, rows, eps, skip); break;
      case 7: launch_k(ln_modulate_v4_kernel<7>, grid, wpb * kWave, 0, s, h, shift, scale, (bf16*)u, rows, eps, skip); break;
      default: launch_k(ln_modulate_v4_kernel<8>, grid, wpb * kWave, 0, s, h, shift, scale, (bf16*)u, rows, eps, skip); break;
    }
  } else if (bf16_out)
    launch_k(ln_modulate_kernel<bf16>, grid, wpb * kWave, 0, s, h, shift, scale, (bf16*)u, rows, D, eps, skip);
  else
    launch_k(ln_modulate_kernel<float>, grid, wpb * kWave, 0, s, h, shift, scale, (float*)u, rows, D, eps, skip);
  return hipGetLastError();
}

template <int VEC, int R, int MAXC, int NW = 8>
void launch_final_t(const FinalArgs& a, hipStream_t s) {
  constexpr int RB = NW * R;
  const int blocks = a.B * ((a.Nv + RB - 1) / RB + (a.Na + RB - 1) / RB);
  if (blocks > 0) launch_k(final_kernel<VEC, R, MAXC, NW>, blocks, NW * 64, 0, s, a);
}

hipError_t launch_final(const FinalArgs& a, hipStream_t s) {
  if (a.D % kWave || a.D > 2048 || a.Cv > kFinalCout || a.A > kFinalCout) return hipErrorInvalidValue;
  // the widest column vector D allows; the smallest LDS copy that holds the
  // weights (48 KB at D <= 768, so that several blocks share a CU); four rows
  // per wave share each weight read (two where the rows' registers would not
  // fit), or one row per wave for short trajectories (under 4096 rows: the
  // small model's 800 rows as 100 blocks of 8)
  const bool many = (long)a.B * (a.Nv + a.Na) >= 4096;
  if (a.D % 256 == 0) {
    if (a.D <= 768)
      many ? launch_final_t<4, 4, 3>(a, s) : launch_final_t<4, 1, 3>(a, s);
    else if (a.D <= 1024)
      many ? launch_final_t<4, 4, 4>(a, s) : launch_final_t<4, 1, 4>(a, s);
    else if (a.D <= 1536)
      many ? launch_final_t<4, 4, 6>(a, s) : launch_final_t<4, 1, 6>(a, s);
    else
      launch_final_t<4, 2, 8>(a, s);
  } else if (a.D % 128 == 0) {
    if (a.D <= 1024)
      many ? launch_final_t<2, 4, 8>(a, s) : launch_final_t<2, 1, 8>(a, s);
    else
      launch_final_t<2, 2, 16>(a, s);
  } else {
    if (a.D <= 1024)
      many ? launch_final_t<1, 4, 16>(a, s) : launch_final_t<1, 1, 16>(a, s);
    else
      launch_final_t<1, 2, 32>(a, s);
  }
  return hipGetLastError();
}

hipError_t launch_rr_gate(const RRGateArgs& a, hipStream_t s) {
  const int rows = a.B * a.T;
  if (a.D % 4) return hipErrorInvalidValue;
  const int wpb = 4;
  if (a.D % 256 == 0 && a.D <= 2048) {
    const int per = (a.T - a.Na + 3) / 4 + (a.Na + 3) / 4;
    launch_k(rr_gate_partials_kernel<8>, (unsigned)(a.B * per), 256, 0, s, a);
    launch_k(rr_gate_finish_kernel, (unsigned)(a.B * 2), 256, 0, s, a);
    return hipGetLastError();
  }
  launch_k(rr_row_sums_kernel, (rows + wpb - 1) / wpb, wpb * kWave, 0, s, a.hs, a.hq, a.pa, a.row_sums, rows, a.D);
  launch_k(rr_finish_kernel, a.B * 2, 1024, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_rr_inject(float* h, const float* Ra, const double* result, int B, int T, int D,
                            int Nv, int Na, hipStream_t s, const int* flag) {
  const int64_t n4 = (int64_t)B * T * D / 4;
  if (D % 4 || n4 >= (int64_t)1 << 31) return hipErrorInvalidValue;
  const unsigned grid = (unsigned)((n4 + 256 * kInjV - 1) / (256 * kInjV));
  launch_k(rr_inject_kernel, grid, 256, 0, s, h, Ra, result, B, T, D, Nv, Na, flag);
  return hipGetLastError();
}

hipError_t launch_rr_pre_middle(const float* h, float* hq, float* pa, int64_t n, hipStream_t s,
                                const int* flag) {
  const int64_t n4 = n / 4;
  launch_k(rr_pre_middle_kernel, (unsigned)((n4 + 255) / 256), 256, 0, s, h, hq, pa, n4, flag);
  return hipGetLastError();
}

hipError_t launch_rr_refresh(const float* h, const float* hq, float* Ra, int64_t n, hipStream_t s,
                             const int* flag) {
  const int64_t n4 = n / 4;
  launch_k(rr_refresh_kernel, (unsigned)((n4 + 255) / 256), 256, 0, s, h, hq, Ra, n4, flag);
  return hipGetLastError();
}

hipError_t launch_rr_decide(const double* result, int B, int nbranch, int force_accept, int* flag,
                            double* hist_stats, int* hist_flag, hipStream_t s) {
  launch_k(rr_decide_kernel, 1, 64, 0, s, result, B, nbranch, force_accept, flag, hist_stats, hist_flag);
  return hipGetLastError();
}

hipError_t launch_pack_condition(const float* obs, int n_obs, int c_obs, const float* ctx, int n_ctx, int c_ctx,
                                 int64_t ctx_stride, float* cond, int B, int Co, hipStream_t s) {
  const int64_t n = (int64_t)B * (n_obs + n_ctx) * Co;
  if (n == 0) return hipSuccess;
  launch_k(pack_condition_kernel, (unsigned)((n + 255) / 256), 256, 0, s, obs, n_obs, c_obs, ctx, n_ctx, c_ctx,
           ctx_stride, cond, B, Co);
  return hipGetLastError();
}

hipError_t launch_copy_f32(const float* src, float* dst, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (n % 4 == 0 && reinterpret_cast<uintptr_t>(src) % 16 == 0 && reinterpret_cast<uintptr_t>(dst) % 16 == 0) {
    const int64_t n4 = n / 4;
    launch_k(copy_f32x4_kernel, (unsigned)((n4 + 1023) / 1024), 256, 0, s, reinterpret_cast<const f32x4*>(src),
             reinterpret_cast<f32x4*>(dst), n4);
  } else {
    launch_k(copy_f32_kernel, (unsigned)((n + 255) / 256), 256, 0, s, src, dst, n);
  }
  return hipGetLastError();
}

namespace {
bool aligned16(const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; }
}  // namespace

hipError_t launch_remap(const RemapArgs& a, hipStream_t s) {
  const int64_t nv = (int64_t)a.Nv * a.Cv, na = (int64_t)a.Na * a.A, traj = nv + na;
  // 16-byte path: every group of four floats starts 16-byte aligned in each
  // array, in its branch and at its shifted source
  const bool sums_vec = aligned16(a.x_r) && aligned16(a.x_bar) && nv % 4 == 0 && na % 4 == 0;
  const bool apply_vec = sums_vec && aligned16(a.noise) && aligned16(a.x_out) &&
                         ((int64_t)a.shift_video * a.Cv) % 4 == 0 && ((int64_t)a.shift_action * a.A) % 4 == 0;
  const int nch = std::max(reduce_chunks(nv), reduce_chunks(na));
  if (sums_vec)
    launch_k(remap_partial_kernel<true>, dim3(nch, a.B * 2), 256, 0, s, a);
  else
    launch_k(remap_partial_kernel<false>, dim3(nch, a.B * 2), 256, 0, s, a);
  launch_k(remap_finish_kernel, a.B * 2, 256, 0, s, a);
  if (apply_vec)
    launch_k(remap_apply_kernel<true>, dim3((unsigned)((traj / 4 + 255) / 256), a.B), 256, 0, s, a);
  else
    launch_k(remap_apply_kernel<false>, dim3((unsigned)((traj + 255) / 256), a.B), 256, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_or_sums(int n_comp, const float* const* u_hat, const float* const* u,
                          const int64_t* n, const double* delta, double* sums, hipStream_t s) {
  if (n_comp < 1 || n_comp > WAM_MAX_COMPONENTS) return hipErrorInvalidValue;
  OrSumArgs a{};
  bool vec = true;
  for (int m = 0; m < n_comp; ++m) {
    a.u_hat[m] = u_hat[m];
    a.u[m] = u[m];
    a.n[m] = n[m];
    a.inv_delta[m] = 1.0 / delta[m];
    vec = vec && aligned16(u_hat[m]) && aligned16(u[m]) && n[m] % 4 == 0;
  }
  a.sums = sums;
  int nch = 1;
  for (int m = 0; m < n_comp; ++m) nch = std::max(nch, reduce_chunks(n[m]));
  if (vec)
    launch_k(or_sums_kernel<true>, dim3(nch, n_comp), 256, 0, s, a);
  else
    launch_k(or_sums_kernel<false>, dim3(nch, n_comp), 256, 0, s, a);
  return hipGetLastError();
}

}  // namespace wam

// ================================================================ no-alloc remap
// Trajectory Remapping for callers that cannot allocate device memory (code
// under graph capture, tight serving loops): the rms and run-sum scratch of
// the remap kernels lives in this file-scope device array instead of a
// workspace.  Each GPU holds its own copy until the process ends; its device
// address is looked up once per device (with that device current) and only
// that address is ever handed to kernels or copies.
namespace wam {
namespace {

constexpr int kNoAllocScratchDoubles = WAM_MAX_BATCH * 2 * (1 + kRemapChunks);  // 256.3 KiB
constexpr int kMaxDevices = 64;

__device__ __align__(256) double scratch[kNoAllocScratchDoubles];

std::mutex g_scratch_mu;
double* g_scratch_ptr[kMaxDevices] = {};

thread_local std::string t_noalloc_err;

int noalloc_fail(int code, const char* msg) {
  t_noalloc_err = msg;
  return code;
}

// Device address of this GPU's copy of `scratch` (looked up on first use).
int scratch_for_current_device(double** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return noalloc_fail(WAM_E_HIP, "wam_remap_noalloc: no current device");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p)
      return noalloc_fail(WAM_E_HIP, "wam_remap_noalloc: hipGetSymbolAddress of the scratch array failed");
    g_scratch_ptr[dev] = static_cast<double*>(p);
  }
  *out = g_scratch_ptr[dev];
  return WAM_OK;
}

}  // namespace
}  // namespace wam

extern "C" {

const char* wam_noalloc_last_error(void) { return wam::t_noalloc_err.c_str(); }

int wam_remap_noalloc(const wam_config* cfg, const wam_remap_args* a, void* hip_stream) {
  using namespace wam;
  if (!cfg || !a) return noalloc_fail(WAM_E_ARG, "wam_remap_noalloc: null argument");
  if (cfg->B < 1 || cfg->B > WAM_MAX_BATCH)
    return noalloc_fail(WAM_E_SHAPE, "wam_remap_noalloc: batch must be 1..WAM_MAX_BATCH (16): the static "
                                     "scratch holds 16 x 2 x 1025 float64 sums");
  if (cfg->Nv < 0 || cfg->Na < 0 || cfg->Cv < 1 || cfg->A < 1 || cfg->Nv + cfg->Na < 1)
    return noalloc_fail(WAM_E_SHAPE, "wam_remap_noalloc: need Nv, Na >= 0, Nv + Na >= 1, Cv, A >= 1");
  const int64_t traj = (int64_t)cfg->Nv * cfg->Cv + (int64_t)cfg->Na * cfg->A;
  if (traj * cfg->B > (int64_t)INT32_MAX)
    return noalloc_fail(WAM_E_SHAPE, "wam_remap_noalloc: B * traj must fit in 31 bits");
  if (!a->x_bar || !a->x_r || !a->noise || !a->x_out)
    return noalloc_fail(WAM_E_ARG, "wam_remap_noalloc: null remap argument");
  if (!(a->sigma_r > 0.f)) return noalloc_fail(WAM_E_ARG, "wam_remap_noalloc: sigma_r must be > 0");
  if (!(a->sigma_b0 >= 0.f)) return noalloc_fail(WAM_E_ARG, "wam_remap_noalloc: sigma_b0 must be >= 0");
  if (a->shift_action < 0 || a->shift_video < 0)
    return noalloc_fail(WAM_E_ARG, "wam_remap_noalloc: shifts must be >= 0");
  if (a->x_out == a->x_bar || a->x_out == a->x_r)
    return noalloc_fail(WAM_E_ARG, "wam_remap_noalloc: x_out must not alias inputs");
  double* sc = nullptr;
  int st = scratch_for_current_device(&sc);
  if (st) return st;
  RemapArgs r{a->x_bar, a->x_r, a->noise, a->x_out, sc, sc + 2 * cfg->B, a->sigma_r, a->sigma_b0,
              a->shift_action, a->shift_video, cfg->B, cfg->Nv, cfg->Cv, cfg->Na, cfg->A};
  if (launch_remap(r, static_cast<hipStream_t>(hip_stream)) != hipSuccess)
    return noalloc_fail(WAM_E_HIP, "wam_remap_noalloc: kernel launch failed");
  return WAM_OK;
}

}  // extern "C"
