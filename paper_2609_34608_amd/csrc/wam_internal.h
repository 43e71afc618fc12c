// Internal declarations shared by the libwam translation units (gfx950 only).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>

#include "wam.h"

namespace wam {

using bf16 = __bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// ---------------------------------------------------------------- launches
// Per-class kernel timing.  While a timing scope is armed (start / stop
// events set), launches go through hipExtLaunchKernel, which stamps the start
// event with the begin of the scope's first dispatch and the stop event with
// the end of each dispatch: the event pair spans exactly the scope's kernels,
// with no event-record packets in between.  Unarmed, a launch is a plain one.
struct LaunchTiming {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
  bool started = false;  // the start event has been attached to a dispatch
};
inline LaunchTiming& launch_timing() {
  static thread_local LaunchTiming t;
  return t;
}
template <typename... KArgs, typename... Args>
inline void launch_k(void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t lds, hipStream_t s, Args... args) {
  LaunchTiming& t = launch_timing();
  if (t.stop) {
    hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)lds, s, t.started ? nullptr : t.start, t.stop, 0u,
                          static_cast<KArgs>(args)...);
    t.started = true;
  } else {
    kernel<<<grid, block, lds, s>>>(static_cast<KArgs>(args)...);
  }
}

// compile-time loop: f(std::integral_constant<int, 0>) ... f(<N-1>); keeps
// register-array indices static after inlining
template <typename F, int... Js>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Js...>) {
  (f(std::integral_constant<int, Js>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// The bf16 QKV epilogue stores q pre-multiplied by log2(e) / sqrt(64), so the
// bf16 attention kernel's scores are already the exponents of exp2.
constexpr float kQLog2Scale = 0.18033688011112042f;  // log2(e) / 8

// Key order inside each 64-key block of the stored V^T rows (bf16 path): key
// 32c + 16h + 4g + r sits at 32c + 8g + 4h + r, so that the eight keys one
// lane feeds to a P.V MFMA (rows 4g..4g+3 of two adjacent 16-key score tiles)
// are adjacent in LDS and load as one 16-byte read.
__host__ __device__ constexpr int vt_key_pos(int k) {
  return (k & 32) | ((k & 12) << 1) | ((k & 16) >> 2) | (k & 3);
}

// ---------------------------------------------------------------- helpers
__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return static_cast<float>(x); }
template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return static_cast<bf16>(x); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// GELU, tanh form: x/2 (1 + tanh(u)), u = sqrt(2/pi)(x + 0.044715 x^3),
// evaluated as x * sigmoid(2u) = x / (1 + 2^(-2u log2 e)) (the same function)
// with the hardware exp2 and reciprocal (v_exp_f32, v_rcp_f32: about 1 ulp)
// instead of a correctly rounded division.  Large |u| saturates: 2^(+inf)
// gives 1/inf = 0, 2^(-inf) gives 1.
__device__ __forceinline__ float gelu_tanh_f(float x) {
  const float c1 = -2.0f * 0.7978845608028654f * 1.4426950408889634f;  // -2 sqrt(2/pi) log2(e)
  const float c3 = c1 * 0.044715f;
  const float z = x * (c1 + c3 * x * x);
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(z));
}

// ---------------------------------------------------------------- GEMM
enum GemmEpilogue : int {
  EPI_BIAS = 0,       // out[m,n] = acc + bias[n]                       (act type)
  EPI_BIAS_GELU = 1,  // out[m,n] = gelu(acc + bias[n])                 (act type)
  EPI_GATED_RES = 2,  // h[m,n] += gate[n] * (acc + bias[n])            (float32)
  EPI_QKV = 3,        // q,k RMS-normalised per head -> [B*H][Tpad][64], v -> [B*H][64][Tpad]
};

// Destination of the QKV epilogue (bf16 mode, head size 64).
struct QkvOut {
  bf16* q;
  bf16* k;
  bf16* vt;
  const float* q_g;
  const float* k_g;
  int T, Tpad, H, D, qk_norm;
  float eps;
};

struct GemmArgs {
  const void* A;     // [M][K] activations (act type), row stride K
  const void* W;     // [N][K] packed weight (act type), row stride K
  const float* bias; // [N]
  const float* gate; // [N] (EPI_GATED_RES)
  void* out;         // [M][N] act type, or float h for EPI_GATED_RES
  int M, N, K;
  int epi;
  int role;          // distinct kernel symbol per projection (0 qkv, 1 proj, 2 fc1, 3 fc2)
  float* partial;    // split-K scratch, splits * M * N floats
  QkvOut qkv;
  const int* skip;   // device flag: when non-null and set, the launch does nothing
  float* copy;       // EPI_GATED_RES: when non-null, the updated h is also stored here ([M][N])
};

struct GemmPlan {
  int cfg;
  int splits;
};

GemmPlan plan_gemm(int M, int N, int K, int epi);
size_t gemm_partial_floats(int M, int N, int K, int epi);
int gemm_num_configs();
hipError_t launch_gemm_cfg(const GemmArgs& a, int cfg, int splits, hipStream_t s);
hipError_t launch_gemm(const GemmArgs& a, bool bf16_mode, hipStream_t s);

// ---------------------------------------------------------------- attention
struct AttnArgs {
  const void* q;   // [B*H][Tpad][dh]
  const void* k;   // [B*H][Tpad][dh]
  const void* vt;  // [B*H][dh][Tpad]
  void* out;       // [B*T][D], head h at columns h*dh
  int B, H, T, Tpad, dh, D;
  const int* skip; // device flag: when non-null and set, the launch does nothing
  // bf16 mode: when bounded is set, every score (log2 units, as the QKV
  // epilogue stores q) lies in [-mref, mref] and the kernel uses mref as its
  // fixed softmax reference
  float mref;
  int bounded;
  int variant;  // WAM_ATTN_*: AUTO picks by shape; bounded forms need bounded set
};
hipError_t launch_attention(const AttnArgs& a, bool bf16_mode, hipStream_t s);
// bf16 kernel forms: running max; and with a.bounded, the fixed reference in
// a software-pipelined loop, a plain loop (also with two wave groups that
// split the keys: 2 nw waves), or the ping-pong form (8 waves in two groups,
// nw ignored)
enum AttnForm : int { ATTN_RUNNING = 0, ATTN_PIPELINED = 1, ATTN_PLAIN = 2, ATTN_PINGPONG = 3, ATTN_PLAIN_KSPLIT = 4 };
// qt query tiles of 16 per wave, nw waves per block, st K / V^T stages
hipError_t launch_attention_cfg(const AttnArgs& a, int qt, int nw, int st, hipStream_t s, int form = ATTN_RUNNING);
// Largest score magnitude, log2 units, that the bf16 QKV epilogue can produce
// for head size 64 with QK-norm gains q_g, k_g (host arrays of 64)
float attention_score_bound(const float* q_g, const float* k_g);

// qkv [B*T][3D] -> q, k (optionally RMS-normalised with gains) and v^T
struct RelayoutArgs {
  const void* qkv;
  const float* q_g;
  const float* k_g;
  void* q;
  void* k;
  void* vt;
  int B, H, T, Tpad, dh, D;
  int qk_norm;
  float eps;
  const int* skip;
};
hipError_t launch_qkv_relayout(const RelayoutArgs& a, bool bf16_mode, hipStream_t s);

// ---------------------------------------------------------------- small kernels
// y[n] = out_act(sum_k in_act(x[k]) W[k][n] + b[n]), W row-major [K][N]
// (float or bf16); act: 0 none, 1 SiLU.  partial: float[ceil(K/kc)][N].
hipError_t launch_gemv(const float* x, const void* W, bool w_bf16, const float* b, float* y,
                       float* partial, int K, int N, int in_act, int out_act, hipStream_t s);
// SiLU(c) with c = SiLU(e(sigma) W1 + b1) W2 + b2, e the 256 sinusoidal features
// (a1: [D] scratch for the hidden layer)
hipError_t launch_timestep_mlp(float sigma, const float* w1, const float* b1, const float* w2, const float* b2,
                               float* a1, float* silu_c, int D, hipStream_t s);

struct EmbedArgs {
  const float* x;     // [B][traj]
  const float* cond;  // [B][No][Co]
  const float* wv; const float* bv;  // [Cv][D], [D]
  const float* wa; const float* ba;  // [A][D], [D]
  const float* wo; const float* bo;  // [Co][D], [D]
  const float* pe;    // [T][D] position embedding
  float* h;           // [B][T][D]
  int B, T, D, Nv, Cv, Na, A, No, Co;
};
hipError_t launch_embed(const EmbedArgs& a, hipStream_t s);

// u = LN(h) * (1 + scale) + shift  (row-wise over D), u in act type
// skip: device flag; when non-null and set the launch does nothing
hipError_t launch_ln_modulate(const float* h, const float* shift, const float* scale, void* u,
                              int rows, int D, float eps, bool bf16_out, hipStream_t s,
                              const int* skip = nullptr);

struct FinalArgs {
  const float* h;      // [B][T][D]
  const float* shift;  // [D]
  const float* scale;  // [D]
  const float* wv; const float* bv;  // head weights transposed [Cv][D], bias [Cv]
  const float* wa; const float* ba;  // [A][D], [A]
  float* v_out;        // [B][traj] or null
  float* x;            // [B][traj] Euler target or null
  float dsigma;        // sigma_{k+1} - sigma_k
  int B, T, D, Nv, Cv, Na, A;
  float eps;
};
hipError_t launch_final(const FinalArgs& a, hipStream_t s);

// Residual Rescaling
struct RRGateArgs {
  const float* hs;   // h_s [M][D]
  const float* hq;   // h_q
  const float* pa;   // retained p_a
  double* row_sums;  // [M][3]: per-row (or per-block) sums p_i p_a, p_i^2, p_a^2
  double* result;    // [B][2][8]: Sip Sii Saa alpha cos fit pass pad
  int B, T, D, Nv, Na;
  float alpha_min, alpha_max, eps, gamma_cos, gamma_fit;
};
hipError_t launch_rr_gate(const RRGateArgs& a, hipStream_t s);
// With a device decision flag (1 = reuse, 0 = refresh) the inject runs only on
// reuse and the pre-middle / refresh passes only on refresh; null = always run.
hipError_t launch_rr_inject(float* h, const float* Ra, const double* result, int B, int T, int D,
                            int Nv, int Na, hipStream_t s, const int* flag = nullptr);
// p_a <- h - hq ; hq <- h   (before recomputing the middle)
hipError_t launch_rr_pre_middle(const float* h, float* hq, float* pa, int64_t n, hipStream_t s,
                                const int* flag = nullptr);
// R_a <- h - hq  (hq holds h_s)
hipError_t launch_rr_refresh(const float* h, const float* hq, float* Ra, int64_t n, hipStream_t s,
                             const int* flag = nullptr);
// Decision on the device: flag = force_accept ? 1 : AND of the (sample, branch)
// pass bits in result over the first nbranch branches; hist_stats [B][2][3]
// (alpha, cos, fit) and hist_flag record the step for a later read-back.
hipError_t launch_rr_decide(const double* result, int B, int nbranch, int force_accept, int* flag,
                            double* hist_stats, int* hist_flag, hipStream_t s);
// cond [B][n_obs + n_ctx][Co]: obs tokens then ctx tokens, zero-padded channels
hipError_t launch_pack_condition(const float* obs, int n_obs, int c_obs, const float* ctx, int n_ctx, int c_ctx,
                                 int64_t ctx_stride, float* cond, int B, int Co, hipStream_t s);
// dst <- src (n floats), a kernel rather than a copy engine command
hipError_t launch_copy_f32(const float* src, float* dst, int64_t n, hipStream_t s);

// Trajectory Remapping
// Chunked float64 reductions (remap rms, rebinding score): a reduction over n
// elements is cut into reduce_chunks(n) runs of equal length (at least
// kReduceRun elements each, at most kRemapChunks runs), one block per run,
// and the run sums are added in run order.
constexpr int kRemapChunks = 1024;
constexpr int kReduceRun = 2048;
__host__ __device__ inline int reduce_chunks(int64_t n) {
  const int64_t c = (n + kReduceRun - 1) / kReduceRun;
  return (int)(c < 1 ? 1 : (c > kRemapChunks ? kRemapChunks : c));
}
struct RemapArgs {
  const float* x_bar; const float* x_r; const float* noise; float* x_out;
  double* coef;     // [B][2] scratch: sigma_b0 / (sigma_r rms) per (sample, branch)
  double* partial;  // [B][2][kRemapChunks] scratch
  float sigma_r, sigma_b0;
  int shift_action, shift_video;
  int B, Nv, Cv, Na, A;
};
hipError_t launch_remap(const RemapArgs& a, hipStream_t s);

// Observation Rebinding: sums of ((u_hat-u)/delta)^2 per component, float64
// run sums [n_comp][kRemapChunks] (the first reduce_chunks(n[m]) of row m)
hipError_t launch_or_sums(int n_comp, const float* const* u_hat, const float* const* u,
                          const int64_t* n, const double* delta, double* sums, hipStream_t s);

}  // namespace wam
