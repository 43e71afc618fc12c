// libwam C ABI: handle, validation, weight packing, workspace carving, the
// denoising-step driver and the joint replan runtime (host side).
#include <math.h>
#include <string.h>

#include <algorithm>
#include <cstdio>
#include <string>
#include <vector>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "wam_internal.h"

using namespace wam;

namespace {

constexpr int kTimeDim = 256;
constexpr size_t kAlign = 256;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

uint16_t f32_to_bf16_bits(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffff) ? 0x40 : 0));
  const uint32_t lsb = (u >> 16) & 1u;
  u += 0x7fffu + lsb;
  return (uint16_t)(u >> 16);
}

struct Dims {
  int B, L, D, H, F, Nv, Cv, Na, A, No, Co, T, M, dh, Tpad, traj, Nmod;
  bool bf;
  size_t act;  // bytes per activation element
};

int make_dims(const wam_config* c, Dims* d, std::string* why) {
  auto bad = [&](const char* m) {
    if (why) *why = m;
    return WAM_E_SHAPE;
  };
  if (!c) {
    if (why) *why = "null config";
    return WAM_E_ARG;
  }
  if (c->B < 1 || c->B > WAM_MAX_BATCH) return bad("B must be in 1..WAM_MAX_BATCH");
  if (c->L < 1 || c->D < 64 || c->H < 1 || c->F < 64) return bad("L, D, H, F out of range");
  if (c->Nv < 0 || c->Na < 0 || c->Nv + c->Na < 1 || c->No < 0 || c->Cv < 1 || c->A < 1 || c->Co < 1)
    return bad("token counts / channels out of range");
  if (c->Cv > 16 || c->A > 16 || c->Co > 64) return bad("Cv and A must be <= 16, Co <= 64");
  if (c->D % c->H) return bad("D must be divisible by H");
  if (c->D % 64 || c->D > 2048) return bad("D must be a multiple of 64 and <= 2048");
  if (c->dtype != WAM_FP32 && c->dtype != WAM_BF16) return bad("dtype must be WAM_FP32 or WAM_BF16");
  const int dh = c->D / c->H;
  if (dh != 32 && dh != 64) return bad("head size D/H must be 32 or 64");
  if (c->dtype == WAM_BF16) {
    if (dh != 64) return bad("bf16 mode needs head size 64");
    if (c->F % 128) return bad("bf16 mode needs F a multiple of 128");
  } else {
    if (c->F % 64) return bad("F must be a multiple of 64");
  }
  if (!(c->ln_eps > 0.f)) return bad("ln_eps must be > 0");
  d->B = c->B; d->L = c->L; d->D = c->D; d->H = c->H; d->F = c->F;
  d->Nv = c->Nv; d->Cv = c->Cv; d->Na = c->Na; d->A = c->A; d->No = c->No; d->Co = c->Co;
  d->T = c->Nv + c->Na + c->No;
  d->M = d->B * d->T;
  d->dh = dh;
  d->Tpad = (d->T + 63) / 64 * 64;
  d->traj = c->Nv * c->Cv + c->Na * c->A;
  d->Nmod = c->L * 6 * c->D + 2 * c->D;
  d->bf = c->dtype == WAM_BF16;
  d->act = d->bf ? 2 : 4;
  return WAM_OK;
}

// ---- canonical host weight layout (see wam.h)
struct HostLayout {
  size_t t_w1, t_b1, t_w2, t_b2, in_wv, in_bv, in_wa, in_ba, in_wo, in_bo;
  size_t layer0, layer_stride;
  size_t mod_w, mod_b, qkv_w, qkv_b, q_g, k_g, proj_w, proj_b, fc1_w, fc1_b, fc2_w, fc2_b;  // in layer
  size_t f_mod_w, f_mod_b, out_wv, out_bv, out_wa, out_ba, total;
};

HostLayout host_layout(const Dims& d) {
  HostLayout h{};
  size_t o = 0;
  auto take = [&](size_t n) {
    size_t r = o;
    o += n;
    return r;
  };
  const size_t D = d.D, F = d.F;
  h.t_w1 = take(kTimeDim * D); h.t_b1 = take(D); h.t_w2 = take(D * D); h.t_b2 = take(D);
  h.in_wv = take((size_t)d.Cv * D); h.in_bv = take(D);
  h.in_wa = take((size_t)d.A * D); h.in_ba = take(D);
  h.in_wo = take((size_t)d.Co * D); h.in_bo = take(D);
  h.layer0 = o;
  size_t l = 0;
  auto ltake = [&](size_t n) {
    size_t r = l;
    l += n;
    return r;
  };
  h.mod_w = ltake(D * 6 * D); h.mod_b = ltake(6 * D);
  h.qkv_w = ltake(D * 3 * D); h.qkv_b = ltake(3 * D);
  h.q_g = ltake(d.dh); h.k_g = ltake(d.dh);
  h.proj_w = ltake(D * D); h.proj_b = ltake(D);
  h.fc1_w = ltake(D * F); h.fc1_b = ltake(F);
  h.fc2_w = ltake(F * D); h.fc2_b = ltake(D);
  h.layer_stride = l;
  o += l * d.L;
  h.f_mod_w = take(D * 2 * D); h.f_mod_b = take(2 * D);
  h.out_wv = take(D * d.Cv); h.out_bv = take(d.Cv);
  h.out_wa = take(D * d.A); h.out_ba = take(d.A);
  h.total = o;
  return h;
}

// ---- device weight layout
struct DevLayout {
  // float32 region
  size_t t_w1, t_b1, t_w2, t_b2, in_wv, in_bv, in_wa, in_ba, in_wo, in_bo;
  size_t bmod;                        // [Nmod] all layers' mod_b then f_mod_b
  size_t lbias0, lbias_stride;        // per layer: qkv_b, proj_b, fc1_b, fc2_b, q_g, k_g
  size_t out_wvT, out_bv, out_waT, out_ba;
  size_t pe;                          // [T][D] sinusoidal position embedding (a constant table)
  // activation-typed region
  size_t wmod;                        // [D][Nmod]
  size_t lw0, lw_stride;              // per layer: qkv_wT [3D][D], proj_wT [D][D], fc1_wT [F][D], fc2_wT [D][F]
  size_t total;
};

DevLayout dev_layout(const Dims& d) {
  DevLayout w{};
  size_t o = 0;
  auto f32 = [&](size_t n) {
    size_t r = o;
    o = align_up(o + n * 4);
    return r;
  };
  const size_t D = d.D, F = d.F;
  w.t_w1 = f32(kTimeDim * D); w.t_b1 = f32(D); w.t_w2 = f32(D * D); w.t_b2 = f32(D);
  w.in_wv = f32((size_t)d.Cv * D); w.in_bv = f32(D);
  w.in_wa = f32((size_t)d.A * D); w.in_ba = f32(D);
  w.in_wo = f32((size_t)d.Co * D); w.in_bo = f32(D);
  w.bmod = f32(d.Nmod);
  w.lbias_stride = align_up((3 * D + D + F + D + 2 * d.dh) * 4);
  w.lbias0 = o;
  o += w.lbias_stride * d.L;
  w.out_wvT = f32(D * d.Cv); w.out_bv = f32(d.Cv);
  w.out_waT = f32(D * d.A); w.out_ba = f32(d.A);
  w.pe = f32((size_t)d.T * D);
  w.wmod = o;
  o = align_up(o + D * d.Nmod * d.act);
  w.lw_stride = align_up((3 * D * D + D * D + F * D + D * F) * d.act);
  w.lw0 = o;
  o += w.lw_stride * d.L;
  w.total = o;
  return w;
}

struct WsLayout {
  size_t h, hq, pa, Ra, u, qkv, q, k, vt, attn, mlp, e, a1, sc, mod, gpart, v;
  size_t x_bar, x_r, x_init, x_work, rr_rows, rr_res, tr_rms, or_sums, gsplit, total;
  size_t rr_flag, hist_stats, hist_flag, cond_buf;
  size_t gpart_floats;
};

WsLayout ws_layout(const Dims& d) {
  WsLayout w{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t r = o;
    o = align_up(o + bytes);
    return r;
  };
  const size_t MD = (size_t)d.M * d.D;
  w.h = take(MD * 4); w.hq = take(MD * 4); w.pa = take(MD * 4); w.Ra = take(MD * 4);
  w.u = take(MD * d.act);
  w.qkv = take(MD * 3 * d.act);
  const size_t head = (size_t)d.B * d.H * d.Tpad * d.dh;
  w.q = take(head * d.act); w.k = take(head * d.act); w.vt = take(head * d.act);
  w.attn = take(MD * d.act);
  w.mlp = take((size_t)d.M * d.F * d.act);
  w.e = take(kTimeDim * 4); w.a1 = take(d.D * 4); w.sc = take(d.D * 4);
  // modulation table of every schedule step (a pure function of sigma_k)
  w.mod = take((size_t)WAM_MAX_STEPS * d.Nmod * 4);
  const size_t kmax = std::max(d.D, kTimeDim);
  const size_t nmax = std::max<size_t>(d.Nmod, d.D);
  w.gpart_floats = ((kmax + 31) / 32) * nmax;
  w.gpart = take(w.gpart_floats * 4);
  const size_t tr = (size_t)d.B * d.traj * 4;
  w.v = take(tr); w.x_bar = take(tr); w.x_r = take(tr); w.x_init = take(tr); w.x_work = take(tr);
  w.rr_rows = take((size_t)d.M * 3 * 8);
  w.rr_res = take((size_t)d.B * 2 * 8 * 8);
  w.tr_rms = take((size_t)d.B * 2 * (1 + kRemapChunks) * 8);  // rms, then the run sums
  w.or_sums = take((size_t)WAM_MAX_COMPONENTS * kRemapChunks * 8);  // run sums per component
  size_t split = 0;
  if (d.bf) {
    split = std::max(split, gemm_partial_floats(d.M, 3 * d.D, d.D, EPI_QKV));
    split = std::max(split, gemm_partial_floats(d.M, d.D, d.D, EPI_GATED_RES));
    split = std::max(split, gemm_partial_floats(d.M, d.F, d.D, EPI_BIAS_GELU));
    split = std::max(split, gemm_partial_floats(d.M, d.D, d.F, EPI_GATED_RES));
  }
  w.gsplit = take(std::max<size_t>(split, 1) * 4);
  // device-side reuse decision: flag and one record per stage
  w.rr_flag = take(4);
  w.hist_stats = take((size_t)WAM_MAX_STEPS * d.B * 2 * 3 * 8);
  w.hist_flag = take((size_t)WAM_MAX_STEPS * 4);
  // condition staging buffer read by captured step graphs
  w.cond_buf = take((size_t)d.B * d.No * d.Co * 4 + 4);
  w.total = o;
  return w;
}

struct ProfSlot {
  bool on = false;
  int max = 0;
  int used = 0;
  std::vector<hipEvent_t> ev;  // 2 per launch
  std::vector<double> work;
};

}  // namespace

struct wam_handle {
  wam_config cfg;
  Dims d;
  DevLayout wl;
  WsLayout ws;
  char* wdev = nullptr;
  char* wsdev = nullptr;
  hipStream_t stream = nullptr;
  std::vector<float> sigmas;
  int K = 0;
  bool layer_valid = false;
  // modulation tables: slot k holds the table of sigma_k once computed; the
  // step being enqueued reads slot mod_k
  bool mod_valid[WAM_MAX_STEPS] = {};
  int mod_k = 0;
  bool has_prev = false;
  int kappa = 0;
  // the condition the retained denoising state continues under (cond_buf):
  // set by WAM_ADAPT_REBIND and by every replan (its real condition)
  bool cond_bound = false;
  double* host_stage = nullptr;  // pinned, 64 KiB
  std::string err;
  ProfSlot prof[WAM_KC_COUNT];
  // per-layer fixed softmax reference (log2 units) of the bf16 attention, or
  // -1 where the scores have no usable bound
  std::vector<float> attn_mref;
  int attn_variant = WAM_ATTN_AUTO;
  bool dev_decision = false;  // RR decision kept on the device (no host round trip per step)
  bool use_graphs = false;    // replay captured step graphs inside wam_replan
  bool capturing = false;
  // captured steps: index k * 3 + variant (0 RR off, 1 establish, 2 attempt)
  std::vector<hipGraphExec_t> graphs;
  wam_rr_profile graph_rr{};
  bool graph_rr_set = false;
  // replan split into begin (remap + anticipatory prefix) and end
  struct Pending {
    bool begun = false;
    bool first = false;   // no retained state: the whole replan runs in end
    bool prefix = false;  // prefix enqueued, its step reports not yet read back
    int entry = 0;
    int nsteps = 0;
    wam_step_info steps[WAM_MAX_STEPS * 2];
    wam_replan_info info;
  } pend;

  template <typename T = float>
  T* W(size_t off) const { return reinterpret_cast<T*>(wdev + off); }
  template <typename T = float>
  T* S(size_t off) const { return reinterpret_cast<T*>(wsdev + off); }
};

namespace {

int fail(wam_t h, int code, const std::string& msg) {
  if (h) h->err = msg;
  return code;
}

#define HIPCHK(h, expr)                                                               \
  do {                                                                                \
    hipError_t e_ = (expr);                                                           \
    if (e_ != hipSuccess)                                                             \
      return fail(h, WAM_E_HIP, std::string(#expr) + ": " + hipGetErrorString(e_));   \
  } while (0)

float* mod_table(wam_t h) { return h->S(h->ws.mod) + (size_t)h->mod_k * h->d.Nmod; }

// roctx range over one phase of a replan or one denoising step (host-side
// annotations for a marker trace; they cost nothing without a profiler).
struct Phase {
  explicit Phase(const char* name) { roctxRangePushA(name); }
  ~Phase() { roctxRangePop(); }
  Phase(const Phase&) = delete;
  Phase& operator=(const Phase&) = delete;
};

// ---- per-launch timing for the measurement API
struct ProfScope {
  wam_t h;
  int kc;
  bool on;
  ProfScope(wam_t h_, int kc_, double work) : h(h_), kc(kc_), on(false) {
    ProfSlot& p = h->prof[kc];
    if (p.on && p.used < p.max && !h->capturing) {
      on = true;
      launch_timing() = LaunchTiming{p.ev[2 * p.used], p.ev[2 * p.used + 1], false};
      p.work[p.used] = work;
    }
  }
  ~ProfScope() {
    if (on) {
      ProfSlot& p = h->prof[kc];
      // a scope whose kernels were all skipped on the host has nothing to time
      if (launch_timing().started) ++p.used;
      launch_timing() = LaunchTiming{};
    }
  }
};

// ---- step pieces
// Modulation table of schedule step k (timestep MLP, then every layer's adaLN
// rows in one GEMV), computed on first use after the schedule is set and read
// by the step's launches from then on; it depends only on sigma_k and the
// weights.  Under capture the computation is recorded but not remembered.
int compute_conditioning(wam_t h, int k) {
  const Dims& d = h->d;
  const DevLayout& wl = h->wl;
  const WsLayout& ws = h->ws;
  hipStream_t s = h->stream;
  h->mod_k = k;
  if (h->mod_valid[k]) return WAM_OK;
  HIPCHK(h, launch_timestep_mlp(h->sigmas[k], h->W(wl.t_w1), h->W(wl.t_b1), h->W(wl.t_w2), h->W(wl.t_b2),
                                h->S(ws.a1), h->S(ws.sc), d.D, s));
  // sc now holds SiLU(c); all adaLN modulations in one pass
  HIPCHK(h, launch_gemv(h->S(ws.sc), h->W<char>(wl.wmod), d.bf, h->W(wl.bmod), mod_table(h),
                        h->S(ws.gpart), d.D, d.Nmod, 0, 0, s));
  if (!h->capturing) h->mod_valid[k] = true;
  return WAM_OK;
}

int embed(wam_t h, const float* x, const float* cond) {
  const Dims& d = h->d;
  const DevLayout& wl = h->wl;
  EmbedArgs a{};
  a.x = x; a.cond = cond;
  a.wv = h->W(wl.in_wv); a.bv = h->W(wl.in_bv);
  a.wa = h->W(wl.in_wa); a.ba = h->W(wl.in_ba);
  a.wo = h->W(wl.in_wo); a.bo = h->W(wl.in_bo);
  a.pe = h->W(wl.pe);
  a.h = h->S(h->ws.h);
  a.B = d.B; a.T = d.T; a.D = d.D; a.Nv = d.Nv; a.Cv = d.Cv; a.Na = d.Na; a.A = d.A; a.No = d.No; a.Co = d.Co;
  HIPCHK(h, launch_embed(a, h->stream));
  return WAM_OK;
}

// copy: when non-null, the layer's MLP-down epilogue (the last writer of h)
// also stores the layer's output h there.
int run_layer(wam_t h, int l, const int* skip = nullptr, float* copy = nullptr) {
  const Dims& d = h->d;
  const DevLayout& wl = h->wl;
  const WsLayout& ws = h->ws;
  hipStream_t s = h->stream;
  const size_t D = d.D;
  const float* mod = mod_table(h) + (size_t)l * 6 * D;
  const float* lb = h->W(wl.lbias0 + wl.lbias_stride * l);
  const float* qkv_b = lb;
  const float* proj_b = lb + 3 * D;
  const float* fc1_b = proj_b + D;
  const float* fc2_b = fc1_b + d.F;
  const float* q_g = fc2_b + D;
  const float* k_g = q_g + d.dh;
  const char* lw = h->W<char>(wl.lw0 + wl.lw_stride * l);
  const char* qkv_w = lw;
  const char* proj_w = qkv_w + 3 * D * D * d.act;
  const char* fc1_w = proj_w + D * D * d.act;
  const char* fc2_w = fc1_w + (size_t)d.F * D * d.act;
  float* hh = h->S(ws.h);
  const double M = d.M;

  HIPCHK(h, launch_ln_modulate(hh, mod + 0 * D, mod + 1 * D, h->S<char>(ws.u), d.M, d.D, h->cfg.ln_eps, d.bf, s,
                               skip));
  {
    ProfScope ps(h, WAM_KC_GEMM_QKV, 2.0 * M * D * 3 * D);
    GemmArgs g{};
    g.A = h->S<char>(ws.u); g.W = qkv_w; g.bias = qkv_b; g.M = d.M; g.N = (int)(3 * D); g.K = (int)D;
    g.role = 0; g.partial = h->S(ws.gsplit); g.skip = skip;
    if (d.bf) {
      // projection with q/k RMS-norm and the head-major relayout fused in
      g.epi = EPI_QKV;
      g.qkv = QkvOut{h->S<bf16>(ws.q), h->S<bf16>(ws.k), h->S<bf16>(ws.vt), q_g, k_g,
                     d.T, d.Tpad, d.H, d.D, h->cfg.qk_norm, h->cfg.ln_eps};
      HIPCHK(h, launch_gemm(g, true, s));
    } else {
      g.epi = EPI_BIAS; g.out = h->S<char>(ws.qkv);
      HIPCHK(h, launch_gemm(g, false, s));
    }
  }
  if (!d.bf) {
    RelayoutArgs r{h->S<char>(ws.qkv), q_g, k_g, h->S<char>(ws.q), h->S<char>(ws.k), h->S<char>(ws.vt),
                   d.B, d.H, d.T, d.Tpad, d.dh, d.D, h->cfg.qk_norm, h->cfg.ln_eps, skip};
    HIPCHK(h, launch_qkv_relayout(r, false, s));
  }
  {
    ProfScope ps(h, WAM_KC_ATTENTION, 4.0 * d.B * (double)d.T * d.T * D);
    AttnArgs at{h->S<char>(ws.q), h->S<char>(ws.k), h->S<char>(ws.vt), h->S<char>(ws.attn),
                d.B, d.H, d.T, d.Tpad, d.dh, d.D, skip};
    at.mref = h->attn_mref[l];
    at.bounded = d.bf && at.mref >= 0.f;
    at.variant = h->attn_variant;
    HIPCHK(h, launch_attention(at, d.bf, s));
  }
  {
    ProfScope ps(h, WAM_KC_GEMM_PROJ, 2.0 * M * D * D);
    GemmArgs g{h->S<char>(ws.attn), proj_w, proj_b, mod + 2 * D, hh, d.M, (int)D, (int)D, EPI_GATED_RES, 1,
               h->S(ws.gsplit), {}, skip};
    HIPCHK(h, launch_gemm(g, d.bf, s));
  }
  HIPCHK(h, launch_ln_modulate(hh, mod + 3 * D, mod + 4 * D, h->S<char>(ws.u), d.M, d.D, h->cfg.ln_eps, d.bf, s,
                               skip));
  {
    ProfScope ps(h, WAM_KC_GEMM_FC1, 2.0 * M * D * d.F);
    GemmArgs g{h->S<char>(ws.u), fc1_w, fc1_b, nullptr, h->S<char>(ws.mlp), d.M, d.F, (int)D, EPI_BIAS_GELU, 2,
               h->S(ws.gsplit), {}, skip};
    HIPCHK(h, launch_gemm(g, d.bf, s));
  }
  {
    ProfScope ps(h, WAM_KC_GEMM_FC2, 2.0 * M * D * d.F);
    GemmArgs g{h->S<char>(ws.mlp), fc2_w, fc2_b, mod + 5 * D, hh, d.M, (int)D, d.F, EPI_GATED_RES, 3,
               h->S(ws.gsplit), {}, skip, copy};
    HIPCHK(h, launch_gemm(g, d.bf, s));
  }
  return WAM_OK;
}

int run_layers(wam_t h, int lo, int hi, const int* skip = nullptr) {
  for (int l = lo; l < hi; ++l) {
    int st = run_layer(h, l, skip);
    if (st) return st;
  }
  return WAM_OK;
}

int check_rr(wam_t h, const wam_rr_profile* rr) {
  if (!rr || rr->mode == WAM_RR_OFF) return WAM_OK;
  if (rr->mode < 0 || rr->mode > WAM_RR_FORCE_FULL) return fail(h, WAM_E_ARG, "unknown RR mode");
  if (!(0 < rr->q && rr->q < rr->s && rr->s < rr->e && rr->e < h->d.L))
    return fail(h, WAM_E_ARG, "RR needs 0 < q < s < e < L");
  if (!(rr->alpha_min <= rr->alpha_max) || !(rr->eps > 0.f))
    return fail(h, WAM_E_ARG, "RR needs alpha_min <= alpha_max and eps > 0");
  if (rr->branches != WAM_RR_JOINT && rr->branches != WAM_RR_SINGLE)
    return fail(h, WAM_E_ARG, "RR branches must be WAM_RR_JOINT or WAM_RR_SINGLE");
  return WAM_OK;
}

// Rows of RR branch 1 as the gate / inject kernels see them: [nv, nv + na)
// is branch 1, every other row branch 0.  A single branch puts all rows in 0.
struct RRRows {
  int nv, na, nbranch;
};
RRRows rr_rows(const Dims& d, const wam_rr_profile* rr) {
  if (rr->branches == WAM_RR_SINGLE) return RRRows{d.T, 0, 1};
  return RRRows{d.Nv, d.Na, 2};
}

// Final layer + heads: velocity into v_out and/or Euler update of x_euler.
int final_step(wam_t h, int k, float* v_out, float* x_euler) {
  const Dims& d = h->d;
  FinalArgs f{};
  const float* fm = mod_table(h) + (size_t)d.L * 6 * d.D;
  f.h = h->S(h->ws.h); f.shift = fm; f.scale = fm + d.D;
  f.wv = h->W(h->wl.out_wvT); f.bv = h->W(h->wl.out_bv);
  f.wa = h->W(h->wl.out_waT); f.ba = h->W(h->wl.out_ba);
  f.v_out = v_out; f.x = x_euler;
  f.dsigma = (k + 1 <= h->K) ? h->sigmas[k + 1] - h->sigmas[k] : 0.f;
  f.B = d.B; f.T = d.T; f.D = d.D; f.Nv = d.Nv; f.Cv = d.Cv; f.Na = d.Na; f.A = d.A; f.eps = h->cfg.ln_eps;
  HIPCHK(h, launch_final(f, h->stream));
  return WAM_OK;
}

// One denoising step with the reuse decision taken on the device: the gate
// writes a flag that the inject (reuse) and the pre-middle / middle-layer /
// refresh launches (refresh) read, so nothing returns to the host.  Every
// launch is enqueued whatever the outcome, which also makes the sequence
// capturable.  attempt: a retained state exists and the mode runs the gate.
int enqueue_step_device(wam_t h, int k, const float* x, const float* cond, float* v_out, float* x_euler,
                        const wam_rr_profile* rr, bool attempt) {
  const Dims& d = h->d;
  const WsLayout& ws = h->ws;
  hipStream_t s = h->stream;
  int st = compute_conditioning(h, k);
  if (st) return st;
  if ((st = embed(h, x, cond))) return st;
  float* hh = h->S(ws.h);
  const int64_t MD = (int64_t)d.M * d.D;
  if (!rr || rr->mode == WAM_RR_OFF) {
    if ((st = run_layers(h, 0, d.L))) return st;
    return final_step(h, k, v_out, x_euler);
  }
  // the head [0, q): the last layer's MLP-down epilogue also writes h_q
  if ((st = run_layers(h, 0, rr->q - 1))) return st;
  if ((st = run_layer(h, rr->q - 1, nullptr, h->S(ws.hq)))) return st;
  if ((st = run_layers(h, rr->q, rr->s))) return st;
  const int* flag = nullptr;
  if (attempt) {
    const RRRows br = rr_rows(d, rr);
    RRGateArgs g{hh, h->S(ws.hq), h->S(ws.pa), h->S<double>(ws.rr_rows), h->S<double>(ws.rr_res),
                 d.B, d.T, d.D, br.nv, br.na, rr->alpha_min, rr->alpha_max, rr->eps, rr->gamma_cos,
                 rr->gamma_fit};
    {
      ProfScope ps(h, WAM_KC_RR_GATE, 3.0 * MD * 4);
      HIPCHK(h, launch_rr_gate(g, s));
    }
    HIPCHK(h, launch_rr_decide(h->S<double>(ws.rr_res), d.B, br.nbranch, rr->mode == WAM_RR_FORCE_SKIP,
                               h->S<int>(ws.rr_flag), h->S<double>(ws.hist_stats) + (size_t)k * d.B * 6,
                               h->S<int>(ws.hist_flag) + k, s));
    flag = h->S<int>(ws.rr_flag);
    {
      ProfScope ps(h, WAM_KC_RR_INJECT, 3.0 * MD * 4);
      HIPCHK(h, launch_rr_inject(hh, h->S(ws.Ra), h->S<double>(ws.rr_res), d.B, d.T, d.D, br.nv, br.na, s, flag));
    }
  }
  HIPCHK(h, launch_rr_pre_middle(hh, h->S(ws.hq), h->S(ws.pa), MD, s, flag));
  if ((st = run_layers(h, rr->s, rr->e, flag))) return st;
  {
    ProfScope ps(h, WAM_KC_RR_REFRESH, 3.0 * MD * 4);
    HIPCHK(h, launch_rr_refresh(hh, h->S(ws.hq), h->S(ws.Ra), MD, s, flag));
  }
  if ((st = run_layers(h, rr->e, d.L))) return st;
  return final_step(h, k, v_out, x_euler);
}

bool same_rr(const wam_rr_profile& a, const wam_rr_profile& b) { return memcmp(&a, &b, sizeof(a)) == 0; }

void drop_graphs(wam_t h) {
  for (auto& g : h->graphs)
    if (g) hipGraphExecDestroy(g);
  h->graphs.clear();
  h->graph_rr_set = false;
}

// Device-decision step, replayed from a captured graph when graphs are on and
// the step reads the internal trajectory / condition buffers (the pointers a
// graph bakes in).  Capture happens on first use of each (stage, variant).
int device_step(wam_t h, int k, const float* x, const float* cond, float* x_euler, const wam_rr_profile* rr,
                bool attempt) {
  const bool graphable = h->use_graphs && x == h->S(h->ws.x_work) && x_euler == x &&
                         cond == h->S(h->ws.cond_buf);
  bool profiling = false;
  for (auto& p : h->prof) profiling = profiling || p.on;
  if (!graphable || profiling) return enqueue_step_device(h, k, x, cond, nullptr, x_euler, rr, attempt);
  const bool active = rr && rr->mode != WAM_RR_OFF;
  if (active && (!h->graph_rr_set || !same_rr(h->graph_rr, *rr))) {
    drop_graphs(h);
    h->graph_rr = *rr;
    h->graph_rr_set = true;
  }
  const int variant = !active ? 0 : (attempt ? 2 : 1);
  const size_t idx = (size_t)k * 3 + variant;
  if (h->graphs.size() < (size_t)h->K * 3) h->graphs.resize((size_t)h->K * 3, nullptr);
  if (!h->graphs[idx]) {
    // the modulation table is computed outside the graph, which only reads it
    int st0 = compute_conditioning(h, k);
    if (st0) return st0;
    hipGraph_t g = nullptr;
    HIPCHK(h, hipStreamBeginCapture(h->stream, hipStreamCaptureModeThreadLocal));
    h->capturing = true;
    int st = enqueue_step_device(h, k, x, cond, nullptr, x_euler, rr, attempt);
    h->capturing = false;
    hipError_t e = hipStreamEndCapture(h->stream, &g);
    if (st) {
      if (g) hipGraphDestroy(g);
      return st;
    }
    if (e != hipSuccess) return fail(h, WAM_E_HIP, std::string("graph capture: ") + hipGetErrorString(e));
    hipGraphExec_t ex = nullptr;
    e = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
    hipGraphDestroy(g);
    if (e != hipSuccess) return fail(h, WAM_E_HIP, std::string("graph instantiate: ") + hipGetErrorString(e));
    h->graphs[idx] = ex;
  }
  HIPCHK(h, hipGraphLaunch(h->graphs[idx], h->stream));
  return WAM_OK;
}

// Full forward with Residual Rescaling, then the final layer (velocity into
// v_out and/or Euler update of x by dsigma).  With the device decision the
// step info is completed later from the per-stage record (read_history).
int forward(wam_t h, int k, const float* x, const float* cond, float* v_out, float* x_euler,
            const wam_rr_profile* rr, wam_step_info* info) {
  const Dims& d = h->d;
  const WsLayout& ws = h->ws;
  hipStream_t s = h->stream;
  wam_step_info local{};
  wam_step_info* in = info ? info : &local;
  memset(in, 0, sizeof(*in));
  in->layers_evaluated = d.L;
  const bool active = rr && rr->mode != WAM_RR_OFF;
  if (h->dev_decision) {
    const bool attempt = active && h->layer_valid && (rr->mode == WAM_RR_AUTO || rr->mode == WAM_RR_FORCE_SKIP);
    in->rr_active = active;
    in->rr_attempted = attempt;
    int st = v_out ? enqueue_step_device(h, k, x, cond, v_out, x_euler, rr, attempt)
                   : device_step(h, k, x, cond, x_euler, rr, attempt);
    if (st) return st;
    if (active) h->layer_valid = true;  // either path leaves a valid retained state
    return WAM_OK;
  }
  int st = compute_conditioning(h, k);
  if (st) return st;
  if ((st = embed(h, x, cond))) return st;
  float* hh = h->S(ws.h);
  const int64_t MD = (int64_t)d.M * d.D;
  if (!active) {
    if ((st = run_layers(h, 0, d.L))) return st;
  } else {
    in->rr_active = 1;
    // the head [0, q): the last layer's MLP-down epilogue also writes h_q
    if ((st = run_layers(h, 0, rr->q - 1))) return st;
    if ((st = run_layer(h, rr->q - 1, nullptr, h->S(ws.hq)))) return st;
    if ((st = run_layers(h, rr->q, rr->s))) return st;
    bool accept = false;
    const RRRows br = rr_rows(d, rr);
    if (h->layer_valid && (rr->mode == WAM_RR_AUTO || rr->mode == WAM_RR_FORCE_SKIP)) {
      in->rr_attempted = 1;
      RRGateArgs g{hh, h->S(ws.hq), h->S(ws.pa), h->S<double>(ws.rr_rows), h->S<double>(ws.rr_res),
                   d.B, d.T, d.D, br.nv, br.na, rr->alpha_min, rr->alpha_max, rr->eps, rr->gamma_cos,
                   rr->gamma_fit};
      {
        ProfScope ps(h, WAM_KC_RR_GATE, 3.0 * MD * 4);
        HIPCHK(h, launch_rr_gate(g, s));
      }
      const size_t nres = (size_t)d.B * 2 * 8;
      HIPCHK(h, hipMemcpyAsync(h->host_stage, h->S<double>(ws.rr_res), nres * 8, hipMemcpyDeviceToHost, s));
      HIPCHK(h, hipStreamSynchronize(s));
      bool all = true;
      for (int b = 0; b < d.B; ++b)
        for (int j = 0; j < 2; ++j) {
          const double* r = h->host_stage + ((size_t)b * 2 + j) * 8;
          const bool live = j < br.nbranch;
          in->alpha[b][j] = live ? r[3] : NAN;
          in->cos[b][j] = live ? r[4] : NAN;
          in->fit[b][j] = live ? r[5] : NAN;
          all = all && (!live || r[6] != 0.0);
        }
      accept = rr->mode == WAM_RR_FORCE_SKIP ? true : all;
    }
    if (accept) {
      ProfScope ps(h, WAM_KC_RR_INJECT, 3.0 * MD * 4);
      HIPCHK(h, launch_rr_inject(hh, h->S(ws.Ra), h->S<double>(ws.rr_res), d.B, d.T, d.D, br.nv, br.na, s));
      in->rr_accepted = 1;
      in->layers_skipped = rr->e - rr->s;
      in->layers_evaluated = d.L - (rr->e - rr->s);
    } else {
      HIPCHK(h, launch_rr_pre_middle(hh, h->S(ws.hq), h->S(ws.pa), MD, s));
      if ((st = run_layers(h, rr->s, rr->e))) return st;
      {
        ProfScope ps(h, WAM_KC_RR_REFRESH, 3.0 * MD * 4);
        HIPCHK(h, launch_rr_refresh(hh, h->S(ws.hq), h->S(ws.Ra), MD, s));
      }
      h->layer_valid = true;
    }
    if ((st = run_layers(h, rr->e, d.L))) return st;
  }
  return final_step(h, k, v_out, x_euler);
}

// Complete the step infos of stages k_from..k_to-1 from the device record
// (one copy and one synchronisation per segment).
int read_history(wam_t h, int k_from, int k_to, const wam_rr_profile* rr, wam_step_info* infos) {
  if (!h->dev_decision || !infos || k_to <= k_from) return WAM_OK;
  const Dims& d = h->d;
  const size_t nst = (size_t)(k_to - k_from) * d.B * 6;
  std::vector<double> stats(nst);
  std::vector<int> flags(k_to - k_from);
  HIPCHK(h, hipMemcpyAsync(stats.data(), h->S<double>(h->ws.hist_stats) + (size_t)k_from * d.B * 6, nst * 8,
                           hipMemcpyDeviceToHost, h->stream));
  HIPCHK(h, hipMemcpyAsync(flags.data(), h->S<int>(h->ws.hist_flag) + k_from, flags.size() * 4,
                           hipMemcpyDeviceToHost, h->stream));
  HIPCHK(h, hipStreamSynchronize(h->stream));
  for (int k = k_from; k < k_to; ++k) {
    wam_step_info& in = infos[k - k_from];
    if (!in.rr_attempted) continue;
    const double* st = stats.data() + (size_t)(k - k_from) * d.B * 6;
    const int nbranch = rr_rows(d, rr).nbranch;
    for (int b = 0; b < d.B; ++b)
      for (int br = 0; br < 2; ++br) {
        const bool live = br < nbranch;
        in.alpha[b][br] = live ? st[(b * 2 + br) * 3 + 0] : NAN;
        in.cos[b][br] = live ? st[(b * 2 + br) * 3 + 1] : NAN;
        in.fit[b][br] = live ? st[(b * 2 + br) * 3 + 2] : NAN;
      }
    if (flags[k - k_from] == 1) {
      in.rr_accepted = 1;
      in.layers_skipped = rr->e - rr->s;
      in.layers_evaluated = d.L - (rr->e - rr->s);
    }
  }
  return WAM_OK;
}

int check_step(wam_t h, int k, const void* x, const void* cond) {
  if (!h) return WAM_E_ARG;
  if (h->pend.begun)
    return fail(h, WAM_E_STATE, "a replan is open (wam_replan_begin without wam_replan_end)");
  if (h->K <= 0) return fail(h, WAM_E_STATE, "schedule not set (wam_set_schedule)");
  if (k < 0 || k >= h->K) return fail(h, WAM_E_ARG, "step index out of range");
  if (!x) return fail(h, WAM_E_ARG, "null trajectory pointer");
  if (!cond && h->d.No > 0) return fail(h, WAM_E_ARG, "null condition pointer and no bound condition");
  return WAM_OK;
}

int copy_traj(wam_t h, float* dst, const float* src) {
  HIPCHK(h, hipMemcpyAsync(dst, src, (size_t)h->d.B * h->d.traj * 4, hipMemcpyDeviceToDevice, h->stream));
  return WAM_OK;
}

// Observation Rebinding's rebinding step (Sec. 3.2): the retained denoising
// state continues under the condition cond, which is copied into the
// handle's condition buffer (stream-ordered).  Nothing else of the retained
// state changes; the layer state persists across the rebinding (Sec. 3.3).
int bind_condition(wam_t h, const float* cond) {
  const Dims& d = h->d;
  float* cb = h->S(h->ws.cond_buf);
  if (d.No > 0 && cond != cb)
    HIPCHK(h, launch_copy_f32(cond, cb, (int64_t)d.B * d.No * d.Co, h->stream));
  h->cond_bound = true;
  return WAM_OK;
}

// A null condition pointer in the step calls means the bound condition.
const float* resolve_cond(wam_t h, const float* cond) {
  if (cond || h->d.No == 0) return cond;
  return h->cond_bound ? h->S(h->ws.cond_buf) : nullptr;
}

// Calls that read or write the retained state while a replan is open
// (between wam_replan_begin and wam_replan_end) would interleave with the
// enqueued anticipatory prefix; they are refused.
int check_not_pending(wam_t h) {
  if (h->pend.begun)
    return fail(h, WAM_E_STATE, "a replan is open (wam_replan_begin without wam_replan_end)");
  return WAM_OK;
}

int continue_impl(wam_t h, int k_from, int k_to, float* x, const float* cond, const wam_rr_profile* rr,
                  int capture_stage, float* x_capture, wam_step_info* infos, bool read_back = true) {
  for (int k = k_from; k < k_to; ++k) {
    if (capture_stage == k && x_capture) {
      int st = copy_traj(h, x_capture, x);
      if (st) return st;
    }
    int st;
    {
      Phase ph("wam: denoising step");
      st = forward(h, k, x, cond, nullptr, x, rr, infos ? &infos[k - k_from] : nullptr);
    }
    if (st) return st;
  }
  if (capture_stage == k_to && x_capture) {
    int st = copy_traj(h, x_capture, x);
    if (st) return st;
  }
  return read_back ? read_history(h, k_from, k_to, rr, infos) : WAM_OK;
}

}  // namespace

// =====================================================================
extern "C" {

const char* wam_status_string(int s) {
  switch (s) {
    case WAM_OK: return "ok";
    case WAM_E_ARG: return "invalid argument";
    case WAM_E_SHAPE: return "unsupported or mismatched shape";
    case WAM_E_STATE: return "invalid state for this call";
    case WAM_E_HIP: return "HIP runtime error";
    case WAM_E_WORKSPACE: return "buffer too small";
    case WAM_E_UNSUPPORTED: return "unsupported";
    default: return "unknown status";
  }
}

size_t wam_host_weight_count(const wam_config* cfg) {
  Dims d;
  if (make_dims(cfg, &d, nullptr)) return 0;
  return host_layout(d).total;
}

size_t wam_weight_bytes(const wam_config* cfg) {
  Dims d;
  if (make_dims(cfg, &d, nullptr)) return 0;
  return dev_layout(d).total;
}

size_t wam_workspace_bytes(const wam_config* cfg) {
  Dims d;
  if (make_dims(cfg, &d, nullptr)) return 0;
  return ws_layout(d).total;
}

int64_t wam_traj_elems(const wam_config* cfg) {
  Dims d;
  if (make_dims(cfg, &d, nullptr)) return 0;
  return d.traj;
}

int wam_init(const wam_config* cfg, const float* hw, size_t n_hw, void* dev_weights, size_t weight_bytes,
             void* dev_ws, size_t ws_bytes, void* stream, wam_t* out) {
  if (!out) return WAM_E_ARG;
  *out = nullptr;
  Dims d;
  std::string why;
  int st = make_dims(cfg, &d, &why);
  if (st) {
    fprintf(stderr, "wam_init: %s\n", why.c_str());
    return st;
  }
  if (!hw || !dev_weights || !dev_ws) return WAM_E_ARG;
  const HostLayout hl = host_layout(d);
  if (n_hw != hl.total) return WAM_E_SHAPE;
  const DevLayout wl = dev_layout(d);
  const WsLayout ws = ws_layout(d);
  if (weight_bytes < wl.total || ws_bytes < ws.total) return WAM_E_WORKSPACE;

  wam_handle* h = new wam_handle();
  h->cfg = *cfg;
  h->d = d;
  h->wl = wl;
  h->ws = ws;
  h->wdev = static_cast<char*>(dev_weights);
  h->wsdev = static_cast<char*>(dev_ws);
  h->stream = static_cast<hipStream_t>(stream);
  // gate statistics (B x 2 x 8 doubles) or the score's run sums (components x runs)
  constexpr size_t kStageBytes = (size_t)WAM_MAX_COMPONENTS * kRemapChunks * 8;
  static_assert(kStageBytes >= (size_t)WAM_MAX_BATCH * 2 * 8 * 8, "host staging size");
  if (hipHostMalloc((void**)&h->host_stage, kStageBytes, hipHostMallocDefault) != hipSuccess) {
    delete h;
    return WAM_E_HIP;
  }

  // ---- pack weights on the host, then one copy
  std::vector<char> buf(wl.total, 0);
  auto f32 = [&](size_t dst, size_t src, size_t n) { memcpy(buf.data() + dst, hw + src, n * 4); };
  const size_t D = d.D, F = d.F;
  f32(wl.t_w1, hl.t_w1, kTimeDim * D); f32(wl.t_b1, hl.t_b1, D);
  f32(wl.t_w2, hl.t_w2, D * D); f32(wl.t_b2, hl.t_b2, D);
  f32(wl.in_wv, hl.in_wv, d.Cv * D); f32(wl.in_bv, hl.in_bv, D);
  f32(wl.in_wa, hl.in_wa, d.A * D); f32(wl.in_ba, hl.in_ba, D);
  f32(wl.in_wo, hl.in_wo, d.Co * D); f32(wl.in_bo, hl.in_bo, D);
  auto put_act = [&](size_t dst_off, size_t idx, float v) {
    if (d.bf) {
      uint16_t b = f32_to_bf16_bits(v);
      memcpy(buf.data() + dst_off + idx * 2, &b, 2);
    } else {
      memcpy(buf.data() + dst_off + idx * 4, &v, 4);
    }
  };
  // transposed copy: src [rows][cols] -> dst [cols][rows]
  auto put_T = [&](size_t dst_off, const float* src, size_t rows, size_t cols) {
    const size_t tb = 64;
    for (size_t r0 = 0; r0 < rows; r0 += tb)
      for (size_t c0 = 0; c0 < cols; c0 += tb)
        for (size_t r = r0; r < std::min(rows, r0 + tb); ++r)
          for (size_t c = c0; c < std::min(cols, c0 + tb); ++c) put_act(dst_off, c * rows + r, src[r * cols + c]);
  };
  for (int l = 0; l < d.L; ++l) {
    const float* L0 = hw + hl.layer0 + hl.layer_stride * l;
    // modulation: rows k of [D][6D] into the shared [D][Nmod] matrix
    for (size_t r = 0; r < D; ++r)
      for (size_t c = 0; c < 6 * D; ++c) put_act(wl.wmod, r * d.Nmod + (size_t)l * 6 * D + c, L0[hl.mod_w + r * 6 * D + c]);
    memcpy(buf.data() + wl.bmod + (size_t)l * 6 * D * 4, L0 + hl.mod_b, 6 * D * 4);
    const size_t lb = wl.lbias0 + wl.lbias_stride * l;
    memcpy(buf.data() + lb, L0 + hl.qkv_b, 3 * D * 4);
    memcpy(buf.data() + lb + 3 * D * 4, L0 + hl.proj_b, D * 4);
    memcpy(buf.data() + lb + 4 * D * 4, L0 + hl.fc1_b, F * 4);
    memcpy(buf.data() + lb + (4 * D + F) * 4, L0 + hl.fc2_b, D * 4);
    memcpy(buf.data() + lb + (5 * D + F) * 4, L0 + hl.q_g, d.dh * 4);
    memcpy(buf.data() + lb + (5 * D + F + d.dh) * 4, L0 + hl.k_g, d.dh * 4);
    float mref = -1.f;
    if (d.bf && cfg->qk_norm) {
      mref = attention_score_bound(L0 + hl.q_g, L0 + hl.k_g);
      if (!(mref <= 60.0f)) mref = -1.f;
    }
    h->attn_mref.push_back(mref);
    const size_t lw = wl.lw0 + wl.lw_stride * l;
    put_T(lw, L0 + hl.qkv_w, D, 3 * D);
    put_T(lw + 3 * D * D * d.act, L0 + hl.proj_w, D, D);
    put_T(lw + 4 * D * D * d.act, L0 + hl.fc1_w, D, F);
    put_T(lw + (4 * D * D + F * D) * d.act, L0 + hl.fc2_w, F, D);
  }
  for (size_t r = 0; r < D; ++r)
    for (size_t c = 0; c < 2 * D; ++c)
      put_act(wl.wmod, r * d.Nmod + (size_t)d.L * 6 * D + c, hw[hl.f_mod_w + r * 2 * D + c]);
  memcpy(buf.data() + wl.bmod + (size_t)d.L * 6 * D * 4, hw + hl.f_mod_b, 2 * D * 4);
  {
    float* wvT = reinterpret_cast<float*>(buf.data() + wl.out_wvT);
    for (size_t r = 0; r < D; ++r)
      for (int c = 0; c < d.Cv; ++c) wvT[(size_t)c * D + r] = hw[hl.out_wv + r * d.Cv + c];
    float* waT = reinterpret_cast<float*>(buf.data() + wl.out_waT);
    for (size_t r = 0; r < D; ++r)
      for (int c = 0; c < d.A; ++c) waT[(size_t)c * D + r] = hw[hl.out_wa + r * d.A + c];
  }
  f32(wl.out_bv, hl.out_bv, d.Cv);
  f32(wl.out_ba, hl.out_ba, d.A);
  {
    // PE[t][i] = sin(t w_i) for i < D/2, cos(t w_{i-D/2}) above, w_j = 10000^(-j/(D/2)),
    // evaluated in double and rounded once
    float* pe = reinterpret_cast<float*>(buf.data() + wl.pe);
    const int half = d.D / 2;
    for (int j = 0; j < half; ++j) {
      const double om = exp(-log(10000.0) * (double)j / (double)half);
      for (int t = 0; t < d.T; ++t) {
        const double ang = (double)t * om;
        pe[(size_t)t * d.D + j] = (float)sin(ang);
        pe[(size_t)t * d.D + half + j] = (float)cos(ang);
      }
    }
  }
  hipError_t e = hipMemcpy(h->wdev, buf.data(), wl.total, hipMemcpyHostToDevice);
  // pads of q/k/v^T beyond T are read by the attention tiles and must be zero
  if (e == hipSuccess) e = hipMemsetAsync(h->wsdev + ws.q, 0, ws.attn - ws.q, h->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(h->stream);
  if (e != hipSuccess) {
    fprintf(stderr, "wam_init: %s\n", hipGetErrorString(e));
    hipHostFree(h->host_stage);
    delete h;
    return WAM_E_HIP;
  }
  *out = h;
  return WAM_OK;
}

void wam_destroy(wam_t h) {
  if (!h) return;
  drop_graphs(h);
  for (auto& p : h->prof)
    for (auto ev : p.ev) hipEventDestroy(ev);
  if (h->host_stage) hipHostFree(h->host_stage);
  delete h;
}

int wam_sync(wam_t h) {
  if (!h) return WAM_E_ARG;
  HIPCHK(h, hipStreamSynchronize(h->stream));
  return WAM_OK;
}

const char* wam_last_error(wam_t h) { return h ? h->err.c_str() : "null handle"; }

int wam_set_option(wam_t h, int option, int value) {
  if (!h) return WAM_E_ARG;
  if (int st_ = check_not_pending(h)) return st_;
  switch (option) {
    case WAM_OPT_DEVICE_DECISION:
      if (!value && h->use_graphs) return fail(h, WAM_E_STATE, "graphs need the device decision");
      h->dev_decision = value != 0;
      return WAM_OK;
    case WAM_OPT_GRAPHS:
      if (value && !h->dev_decision) return fail(h, WAM_E_STATE, "graphs need the device decision");
      if (value && h->stream == nullptr) return fail(h, WAM_E_UNSUPPORTED, "graphs need a non-default stream");
      if (!value) drop_graphs(h);
      h->use_graphs = value != 0;
      return WAM_OK;
    case WAM_OPT_ATTENTION:
      if (value < WAM_ATTN_AUTO || value > WAM_ATTN_PLAIN) return fail(h, WAM_E_ARG, "unknown attention kernel");
      if (value != h->attn_variant) drop_graphs(h);  // captured launches name the kernel
      h->attn_variant = value;
      return WAM_OK;
    default:
      return fail(h, WAM_E_ARG, "unknown option");
  }
}

int wam_set_schedule(wam_t h, const float* sigmas, int K) {
  if (!h) return WAM_E_ARG;
  if (int st_ = check_not_pending(h)) return st_;
  if (!sigmas || K < 1 || K > WAM_MAX_STEPS) return fail(h, WAM_E_ARG, "need 1 <= K <= WAM_MAX_STEPS");
  for (int i = 0; i < K; ++i)
    if (!(sigmas[i + 1] < sigmas[i])) return fail(h, WAM_E_ARG, "sigmas must decrease strictly");
  h->sigmas.assign(sigmas, sigmas + K + 1);
  h->K = K;
  for (bool& v : h->mod_valid) v = false;
  drop_graphs(h);  // captured steps bake the noise levels in
  return WAM_OK;
}

int wam_velocity(wam_t h, int k, const float* x, const float* cond, float* v_out, const wam_rr_profile* rr,
                 wam_step_info* info) {
  if (h) cond = resolve_cond(h, cond);
  int st = check_step(h, k, x, cond);
  if (st) return st;
  if (!v_out) return fail(h, WAM_E_ARG, "null v_out");
  if ((st = check_rr(h, rr))) return st;
  if ((st = forward(h, k, x, cond, v_out, nullptr, rr, info))) return st;
  return read_history(h, k, k + 1, rr, info);
}

int wam_denoise_step(wam_t h, int k, float* x, const float* cond, const wam_rr_profile* rr, wam_step_info* info) {
  if (h) cond = resolve_cond(h, cond);
  int st = check_step(h, k, x, cond);
  if (st) return st;
  if ((st = check_rr(h, rr))) return st;
  if ((st = forward(h, k, x, cond, nullptr, x, rr, info))) return st;
  return read_history(h, k, k + 1, rr, info);
}

int wam_continue(wam_t h, int k_from, int k_to, float* x, const float* cond, const wam_rr_profile* rr,
                 int capture_stage, float* x_capture, wam_step_info* infos) {
  if (!h) return WAM_E_ARG;
  cond = resolve_cond(h, cond);
  int st0 = check_not_pending(h);
  if (st0) return st0;
  if (h->K <= 0) return fail(h, WAM_E_STATE, "schedule not set (wam_set_schedule)");
  if (k_from < 0 || k_to > h->K || k_from > k_to) return fail(h, WAM_E_ARG, "need 0 <= k_from <= k_to <= K");
  if (!x) return fail(h, WAM_E_ARG, "null trajectory pointer");
  if (!cond && h->d.No > 0) return fail(h, WAM_E_ARG, "null condition pointer and no bound condition");
  int st = check_rr(h, rr);
  if (st) return st;
  return continue_impl(h, k_from, k_to, x, cond, rr, capture_stage, x_capture, infos);
}

int wam_hidden(wam_t h, int k, const float* x, const float* cond, int n_layers, float* h_out) {
  if (h) cond = resolve_cond(h, cond);
  int st = check_step(h, k, x, cond);
  if (st) return st;
  if (!h_out || n_layers < 0 || n_layers > h->d.L) return fail(h, WAM_E_ARG, "need 0 <= n_layers <= L");
  if ((st = compute_conditioning(h, k))) return st;
  if ((st = embed(h, x, cond))) return st;
  if ((st = run_layers(h, 0, n_layers))) return st;
  HIPCHK(h, hipMemcpyAsync(h_out, h->S(h->ws.h), (size_t)h->d.M * h->d.D * 4, hipMemcpyDeviceToDevice, h->stream));
  return WAM_OK;
}

int wam_adapt_state(wam_t h, int op, const void* args) {
  if (!h) return WAM_E_ARG;
  const Dims& d = h->d;
  if (op != WAM_ADAPT_RESET_ALL) {
    int st = check_not_pending(h);
    if (st) return st;
  }
  switch (op) {
    case WAM_ADAPT_REMAP: {
      const wam_remap_args* a = static_cast<const wam_remap_args*>(args);
      if (!a || !a->x_bar || !a->x_r || !a->noise || !a->x_out) return fail(h, WAM_E_ARG, "null remap argument");
      if (!(a->sigma_r > 0.f)) return fail(h, WAM_E_ARG, "sigma_r must be > 0");
      if (!(a->sigma_b0 >= 0.f)) return fail(h, WAM_E_ARG, "sigma_b0 must be >= 0");
      if (a->shift_action < 0 || a->shift_video < 0) return fail(h, WAM_E_ARG, "shifts must be >= 0");
      if (a->x_out == a->x_bar || a->x_out == a->x_r) return fail(h, WAM_E_ARG, "x_out must not alias inputs");
      RemapArgs r{a->x_bar, a->x_r, a->noise, a->x_out, h->S<double>(h->ws.tr_rms),
                  h->S<double>(h->ws.tr_rms) + 2 * d.B, a->sigma_r, a->sigma_b0,
                  a->shift_action, a->shift_video, d.B, d.Nv, d.Cv, d.Na, d.A};
      HIPCHK(h, launch_remap(r, h->stream));
      return WAM_OK;
    }
    case WAM_ADAPT_REBIND: {
      const wam_rebind_args* a = static_cast<const wam_rebind_args*>(args);
      if (!a || (!a->cond && d.No > 0)) return fail(h, WAM_E_ARG, "null rebind condition");
      return bind_condition(h, a->cond);
    }
    case WAM_ADAPT_RESET_LAYER:
      h->layer_valid = false;
      return WAM_OK;
    case WAM_ADAPT_RESET_ALL:
      h->layer_valid = false;
      h->has_prev = false;
      h->kappa = 0;
      h->cond_bound = false;
      h->pend.begun = false;
      return WAM_OK;
    case WAM_ADAPT_SET_REPLAN: {
      const wam_replan_state_args* a = static_cast<const wam_replan_state_args*>(args);
      if (!a || !a->x_bar || !a->x_r || a->kappa < 0) return fail(h, WAM_E_ARG, "bad replan state");
      int st = copy_traj(h, h->S(h->ws.x_bar), a->x_bar);
      if (!st) st = copy_traj(h, h->S(h->ws.x_r), a->x_r);
      if (st) return st;
      h->kappa = a->kappa;
      h->has_prev = true;
      return WAM_OK;
    }
    default:
      return fail(h, WAM_E_ARG, "unknown adapt op");
  }
}

int wam_consistency_score(wam_t h, int n, const float* const* u_hat, const float* const* u, const int64_t* cnt,
                          const double* delta, const double* weight, double* S_out) {
  if (!h) return WAM_E_ARG;
  if (int st_ = check_not_pending(h)) return st_;
  if (n < 1 || n > WAM_MAX_COMPONENTS || !u_hat || !u || !cnt || !delta || !weight || !S_out)
    return fail(h, WAM_E_ARG, "bad consistency-score arguments");
  double wsum = 0.0;
  for (int m = 0; m < n; ++m) {
    if (!u_hat[m] || !u[m] || cnt[m] < 1 || !(delta[m] > 0.0) || !(weight[m] >= 0.0))
      return fail(h, WAM_E_ARG, "component needs data, n >= 1, delta > 0, weight >= 0");
    wsum += weight[m];
  }
  if (!(wsum > 0.0)) return fail(h, WAM_E_ARG, "weights sum to zero");
  double* sums = h->S<double>(h->ws.or_sums);
  HIPCHK(h, launch_or_sums(n, u_hat, u, cnt, delta, sums, h->stream));
  HIPCHK(h, hipMemcpyAsync(h->host_stage, sums, (size_t)n * kRemapChunks * 8, hipMemcpyDeviceToHost, h->stream));
  HIPCHK(h, hipStreamSynchronize(h->stream));
  double acc = 0.0;
  for (int m = 0; m < n; ++m) {
    double sm = 0.0;  // the component's run sums, in run order
    const double* runs = h->host_stage + (size_t)m * kRemapChunks;
    for (int c = 0; c < reduce_chunks(cnt[m]); ++c) sm += runs[c];
    const double e2 = sm / (double)cnt[m];  // e_m^2
    acc += weight[m] * e2;
  }
  *S_out = sqrt(acc / wsum);
  return WAM_OK;
}

int wam_pack_condition(wam_t h, const float* obs, int n_obs, int c_obs, const float* ctx, int n_ctx, int c_ctx,
                       int64_t ctx_stride, float* cond) {
  if (!h) return WAM_E_ARG;
  const Dims& d = h->d;
  if (n_obs < 0 || n_ctx < 0 || n_obs + n_ctx != d.No)
    return fail(h, WAM_E_SHAPE, "pack_condition needs n_obs + n_ctx == No");
  if (c_obs < 1 || c_ctx < 1 || c_obs > d.Co || c_ctx > d.Co)
    return fail(h, WAM_E_SHAPE, "pack_condition needs 1 <= c_obs, c_ctx <= Co");
  if ((n_obs > 0 && !obs) || (n_ctx > 0 && !ctx) || (d.No > 0 && !cond))
    return fail(h, WAM_E_ARG, "pack_condition: null buffer");
  if (n_ctx > 0 && ctx_stride < (int64_t)n_ctx * c_ctx)
    return fail(h, WAM_E_ARG, "pack_condition: ctx_stride smaller than n_ctx * c_ctx");
  HIPCHK(h, launch_pack_condition(obs, n_obs, c_obs, ctx, n_ctx, c_ctx, ctx_stride, cond, d.B, d.Co, h->stream));
  return WAM_OK;
}

}  // extern "C"

namespace {

int check_replan_args(wam_t h, const wam_replan_args* a) {
  if (!a || (!a->cond_real && h->d.No > 0) || !a->x_out || !a->noise_remap)
    return fail(h, WAM_E_ARG, "null replan argument");
  if (h->K <= 0) return fail(h, WAM_E_STATE, "schedule not set (wam_set_schedule)");
  const int K = h->K;
  if (a->b0 < 0 || a->b0 >= K) return fail(h, WAM_E_ARG, "need 0 <= b0 < K");
  if (a->tr_enabled && !(a->b0 <= a->r && a->r < K)) return fail(h, WAM_E_ARG, "need b0 <= r < K");
  if (!a->tr_enabled && !(0 <= a->r && a->r < K)) return fail(h, WAM_E_ARG, "need 0 <= r < K");
  const int entry = a->tr_enabled ? a->b0 : 0;
  if (a->or_enabled) {
    if (!(0 < a->k1 && a->k1 < K - entry)) return fail(h, WAM_E_ARG, "need 0 < k1 < K - b0");
    if (!a->cond_pred && h->d.No > 0) return fail(h, WAM_E_ARG, "rebinding needs cond_pred");
    if (a->kappa_max < 0) return fail(h, WAM_E_ARG, "kappa_max must be >= 0");
  }
  if (a->rr.mode != WAM_RR_OFF) {
    int st = check_rr(h, &a->rr);
    if (st) return st;
  }
  if (!h->has_prev && !a->noise_first) return fail(h, WAM_E_ARG, "first replan needs noise_first");
  return WAM_OK;
}

// Steps k0..k1-1 on the working trajectory, recording their reports in the
// pending replan; the latent at the retained stage r is captured on the way.
int run_segment(wam_t h, const wam_replan_args* a, int k0, int k1, const float* cond, bool rr_allowed,
                bool read_back) {
  const Dims& d = h->d;
  const wam_rr_profile* rr = (rr_allowed && a->rr.mode != WAM_RR_OFF) ? &a->rr : nullptr;
  if (h->use_graphs) {  // captured steps read the condition from the handle's buffer
    int st = bind_condition(h, cond);
    if (st) return st;
    cond = h->S(h->ws.cond_buf);
  }
  int st = continue_impl(h, k0, k1, h->S(h->ws.x_work), cond, rr, a->r, h->S(h->ws.x_r),
                         h->pend.steps + h->pend.nsteps, read_back);
  h->pend.nsteps += k1 - k0;
  return st;
}

}  // namespace

extern "C" {

int wam_replan_begin(wam_t h, const wam_replan_args* a) {
  if (!h) return WAM_E_ARG;
  int st = check_replan_args(h, a);
  if (st) return st;
  if (h->pend.begun) return fail(h, WAM_E_STATE, "replan already begun (call wam_replan_end)");
  auto& p = h->pend;
  p.first = p.prefix = false;
  p.nsteps = 0;
  memset(&p.info, 0, sizeof(p.info));
  p.info.S = -1.0;
  for (int i = 0; i < WAM_MAX_STEPS; ++i) p.info.decision[i] = -1;
  p.entry = a->tr_enabled ? a->b0 : 0;
  h->layer_valid = false;  // layer state is scoped to one replan
  p.begun = true;
  if (!h->has_prev) {
    p.first = true;  // nothing to anticipate without a previous replan
    return WAM_OK;
  }
  const Dims& d = h->d;
  float* x_init = h->S(h->ws.x_init);
  Phase ph_begin("wam_replan_begin: remap + anticipatory prefix");
  if (a->tr_enabled) {
    RemapArgs r{h->S(h->ws.x_bar), h->S(h->ws.x_r), a->noise_remap, x_init, h->S<double>(h->ws.tr_rms),
                h->S<double>(h->ws.tr_rms) + 2 * d.B,
                h->sigmas[a->r], h->sigmas[a->b0], a->shift_action, a->shift_video, d.B, d.Nv, d.Cv, d.Na, d.A};
    HIPCHK(h, launch_remap(r, h->stream));
  } else {
    if ((st = copy_traj(h, x_init, a->noise_remap))) return st;
  }
  if ((st = copy_traj(h, h->S(h->ws.x_work), x_init))) return st;
  if (a->or_enabled && h->kappa < a->kappa_max) {
    p.info.n_start = 1;
    p.prefix = true;
    if ((st = run_segment(h, a, p.entry, p.entry + a->k1, a->cond_pred, a->rr_prefix, false))) return st;
  }
  return WAM_OK;
}

int wam_replan_end(wam_t h, const wam_replan_args* a, wam_replan_info* info) {
  if (!h) return WAM_E_ARG;
  int st;
  if (!h->pend.begun && (st = wam_replan_begin(h, a))) return st;
  if ((st = check_replan_args(h, a))) return st;
  auto& p = h->pend;
  p.begun = false;
  const Dims& d = h->d;
  const int K = h->K;
  float* xw = h->S(h->ws.x_work);
  wam_replan_info* inf = &p.info;
  if (p.first) {
    Phase ph("wam_replan_end: first replan (native)");
    if ((st = copy_traj(h, xw, a->noise_first))) return st;
    if ((st = run_segment(h, a, 0, K, a->cond_real, a->rr_first, true))) return st;
    inf->path = WAM_PATH_FIRST;
  } else if (p.prefix) {
    const wam_rr_profile* rrp = (a->rr_prefix && a->rr.mode != WAM_RR_OFF) ? &a->rr : nullptr;
    if ((st = read_history(h, p.entry, p.entry + a->k1, rrp, p.steps))) return st;
    double S = 0.0;
    {
      Phase ph("wam_replan_end: consistency score");
      st = wam_consistency_score(h, a->n_components, a->u_hat, a->u, a->n, a->delta, a->weight, &S);
    }
    if (st) return st;
    inf->S = S;
    if (S < a->tau && h->kappa < a->kappa_max) {
      h->kappa += 1;
      inf->n_bind = 1;
      inf->path = WAM_PATH_ACCEPT;
      Phase ph("wam_replan_end: rebind + continuation");
      if ((st = bind_condition(h, a->cond_real))) return st;
      if ((st = run_segment(h, a, p.entry + a->k1, K, resolve_cond(h, nullptr), a->rr_prefix, true)))
        return st;
    } else {
      h->kappa = 0;
      inf->path = WAM_PATH_REJECT;
      Phase ph("wam_replan_end: restart from the remapped initialisation");
      h->layer_valid = false;
      if ((st = copy_traj(h, xw, h->S(h->ws.x_init)))) return st;
      if ((st = run_segment(h, a, p.entry, K, a->cond_real, a->rr_refresh, true))) return st;
    }
  } else {
    inf->path = a->or_enabled ? WAM_PATH_FORCED : WAM_PATH_DIRECT;
    Phase ph("wam_replan_end: refresh under the real condition");
    if (a->or_enabled) h->kappa = 0;
    if ((st = run_segment(h, a, p.entry, K, a->cond_real, a->rr_refresh, true))) return st;
  }
  if ((st = copy_traj(h, h->S(h->ws.x_bar), xw))) return st;
  if ((st = copy_traj(h, a->x_out, xw))) return st;
  if (inf->path != WAM_PATH_ACCEPT && (st = bind_condition(h, a->cond_real))) return st;
  h->has_prev = true;
  inf->kappa = h->kappa;
  inf->steps = p.nsteps;
  for (int i = 0; i < p.nsteps; ++i) {
    const wam_step_info& s = p.steps[i];
    if (i < WAM_MAX_STEPS) inf->decision[i] = s.rr_attempted ? (int8_t)s.rr_accepted : (int8_t)-1;
    inf->rr_attempts += s.rr_attempted;
    inf->rr_reuses += s.rr_accepted;
    inf->layers_skipped += s.layers_skipped;
    if (s.rr_active) inf->layers_dense += d.L;
  }
  if (info) *info = *inf;
  return WAM_OK;
}

int wam_replan(wam_t h, const wam_replan_args* a, wam_replan_info* info) {
  if (!h) return WAM_E_ARG;
  int st = wam_replan_begin(h, a);
  if (st) return st;
  return wam_replan_end(h, a, info);
}

int wam_get_replan_state(wam_t h, float* xb, float* xr, int32_t* kappa) {
  if (!h) return WAM_E_ARG;
  if (int st_ = check_not_pending(h)) return st_;
  if (!h->has_prev) return fail(h, WAM_E_STATE, "no replan state yet");
  int st;
  if (xb && (st = copy_traj(h, xb, h->S(h->ws.x_bar)))) return st;
  if (xr && (st = copy_traj(h, xr, h->S(h->ws.x_r)))) return st;
  if (kappa) *kappa = h->kappa;
  return WAM_OK;
}

int wam_profile_enable(wam_t h, int kc, int enable, int max_launches) {
  if (!h) return WAM_E_ARG;
  if (kc < 0 || kc >= WAM_KC_COUNT) return fail(h, WAM_E_ARG, "unknown kernel class");
  ProfSlot& p = h->prof[kc];
  if (!enable) {
    p.on = false;
    return WAM_OK;
  }
  if (max_launches < 1) return fail(h, WAM_E_ARG, "max_launches must be >= 1");
  HIPCHK(h, hipStreamSynchronize(h->stream));
  for (auto ev : p.ev) hipEventDestroy(ev);
  p.ev.assign(2 * (size_t)max_launches, nullptr);
  for (auto& ev : p.ev) HIPCHK(h, hipEventCreate(&ev));
  p.work.assign(max_launches, 0.0);
  p.max = max_launches;
  p.used = 0;
  p.on = true;
  return WAM_OK;
}

int wam_profile_read(wam_t h, int kc, double* total_ms, int64_t* launches, double* work) {
  if (!h) return WAM_E_ARG;
  if (kc < 0 || kc >= WAM_KC_COUNT) return fail(h, WAM_E_ARG, "unknown kernel class");
  HIPCHK(h, hipStreamSynchronize(h->stream));
  ProfSlot& p = h->prof[kc];
  double t = 0.0, w = 0.0;
  for (int i = 0; i < p.used; ++i) {
    float ms = 0.f;
    HIPCHK(h, hipEventElapsedTime(&ms, p.ev[2 * i], p.ev[2 * i + 1]));
    t += ms;
    w += p.work[i];
  }
  if (total_ms) *total_ms = t;
  if (launches) *launches = p.used;
  if (work) *work = w;
  return WAM_OK;
}

}  // extern "C"
