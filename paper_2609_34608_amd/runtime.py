"""Python binding of libwam with the same entry points as the C ABI.

PyTorch only provides device memory and the HIP stream; every step of the
denoising path and of the adaptation operators runs in libwam's kernels.
"""
from __future__ import annotations

import ctypes as C
from dataclasses import dataclass

import numpy as np
import torch

from . import _lib as abi


class WamError(RuntimeError):
    pass


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, torch.Tensor):
        if not t.is_cuda:
            raise WamError("libwam takes device tensors only")
        if t.dtype != torch.float32 or not t.is_contiguous():
            raise WamError("device tensors must be contiguous float32")
        return C.c_void_p(t.data_ptr())
    return C.c_void_p(int(t))


def host_weight_order(n_layers: int) -> list[str]:
    """Names of the canonical host weight buffer, in the order wam.h documents."""
    names = ["t_w1", "t_b1", "t_w2", "t_b2", "in_wv", "in_bv", "in_wa", "in_ba", "in_wo", "in_bo"]
    for l in range(n_layers):
        names += [f"l{l}.{n}" for n in ("mod_w", "mod_b", "qkv_w", "qkv_b", "q_g", "k_g", "proj_w",
                                        "proj_b", "fc1_w", "fc1_b", "fc2_w", "fc2_b")]
    names += ["f_mod_w", "f_mod_b", "out_wv", "out_bv", "out_wa", "out_ba"]
    return names


def make_config(B, L, D, H, F, Nv, Cv, Na, A, No, Co, dtype="bf16", qk_norm=True, ln_eps=1e-6) -> abi.WamConfig:
    return abi.WamConfig(B=B, L=L, D=D, H=H, F=F, Nv=Nv, Cv=Cv, Na=Na, A=A, No=No, Co=Co,
                       dtype=abi.WAM_BF16 if dtype == "bf16" else abi.WAM_FP32, qk_norm=int(bool(qk_norm)),
                       ln_eps=ln_eps)


def config_of(spec) -> abi.WamConfig:
    """Config from any object exposing the model fields (B, L, D, ...)."""
    return make_config(spec.B, spec.L, spec.D, spec.H, spec.F, spec.Nv, spec.Cv, spec.Na, spec.A,
                       spec.No, spec.Co, spec.dtype, spec.qk_norm, spec.ln_eps)


def rr_profile(q=0, s=0, e=0, mode=abi.WAM_RR_OFF, alpha_min=1.0, alpha_max=1.25, eps=1e-8,
               gamma_cos=0.80, gamma_fit=0.60, branches=abi.WAM_RR_JOINT) -> abi.WamRRProfile:
    return abi.WamRRProfile(q=q, s=s, e=e, mode=mode, alpha_min=alpha_min, alpha_max=alpha_max, eps=eps,
                          gamma_cos=gamma_cos, gamma_fit=gamma_fit, branches=branches)


@dataclass
class StepInfo:
    rr_active: bool
    attempted: bool
    accepted: bool
    layers_evaluated: int
    layers_skipped: int
    alpha: np.ndarray
    cos: np.ndarray
    fit: np.ndarray

    @classmethod
    def of(cls, s: abi.WamStepInfo, B: int) -> "StepInfo":
        a = np.array([[s.alpha[b][i] for i in range(2)] for b in range(B)])
        c = np.array([[s.cos[b][i] for i in range(2)] for b in range(B)])
        f = np.array([[s.fit[b][i] for i in range(2)] for b in range(B)])
        return cls(bool(s.rr_active), bool(s.rr_attempted), bool(s.rr_accepted), s.layers_evaluated,
                   s.layers_skipped, a, c, f)


class WamModel:
    """One libwam handle with its device weights and workspace (torch-owned)."""

    def __init__(self, cfg: abi.WamConfig, weights: dict, device="cuda", stream: torch.cuda.Stream | None = None,
                 own_stream: bool = False):
        if not torch.cuda.is_available():
            raise WamError("libwam needs a HIP device")
        self.lib = abi.lib()
        self.cfg = cfg
        self.device = torch.device(device)
        self.B = cfg.B
        self.traj = int(self.lib.wam_traj_elems(C.byref(cfg)))
        n_host = int(self.lib.wam_host_weight_count(C.byref(cfg)))
        wbytes = int(self.lib.wam_weight_bytes(C.byref(cfg)))
        wsbytes = int(self.lib.wam_workspace_bytes(C.byref(cfg)))
        if n_host == 0 or wbytes == 0:
            raise WamError("invalid configuration")
        host = np.concatenate([np.ascontiguousarray(weights[n], np.float32).ravel()
                               for n in host_weight_order(cfg.L)])
        if host.size != n_host:
            raise WamError(f"weight count {host.size} != {n_host}")
        if own_stream:  # a dedicated (default-priority) stream, required for graph replay
            stream = torch.cuda.Stream(self.device)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        self.wdev = torch.empty(wbytes, dtype=torch.uint8, device=self.device)
        self.ws = torch.empty(wsbytes, dtype=torch.uint8, device=self.device)
        h = C.c_void_p()
        st = self.lib.wam_init(C.byref(cfg), host.ctypes.data_as(C.c_void_p), host.size,
                               C.c_void_p(self.wdev.data_ptr()), wbytes, C.c_void_p(self.ws.data_ptr()),
                               wsbytes, C.c_void_p(self.stream.cuda_stream), C.byref(h))
        if st != abi.WAM_OK:
            raise WamError(f"wam_init failed: {self.lib.wam_status_string(st).decode()}")
        self.h = h
        self.K = 0

    # ------------------------------------------------------------ helpers
    def _enter(self):
        """Order the handle's stream after torch's current stream (inputs)."""
        cur = torch.cuda.current_stream(self.device)
        if cur.cuda_stream != self.stream.cuda_stream:
            self.stream.wait_stream(cur)

    def _leave(self):
        """Order torch's current stream after the handle's stream (outputs)."""
        cur = torch.cuda.current_stream(self.device)
        if cur.cuda_stream != self.stream.cuda_stream:
            cur.wait_stream(self.stream)

    def _check(self, st, what):
        if st != abi.WAM_OK:
            msg = self.lib.wam_last_error(self.h).decode()
            raise WamError(f"{what}: {self.lib.wam_status_string(st).decode()}: {msg}")

    def close(self):
        if getattr(self, "h", None):
            self.lib.wam_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def new_traj(self):
        return torch.empty((self.B, self.traj), dtype=torch.float32, device=self.device)

    # ------------------------------------------------------------ ABI
    def set_schedule(self, sigmas):
        s = np.ascontiguousarray(sigmas, np.float32)
        self._check(self.lib.wam_set_schedule(self.h, s.ctypes.data_as(C.POINTER(C.c_float)), s.size - 1),
                    "wam_set_schedule")
        self.K = s.size - 1

    def velocity(self, k, x, cond, v_out=None, rr=None):
        self._enter()
        v_out = self.new_traj() if v_out is None else v_out
        info = abi.WamStepInfo()
        self._check(self.lib.wam_velocity(self.h, k, _ptr(x), _ptr(cond), _ptr(v_out),
                                          C.byref(rr) if rr is not None else None, C.byref(info)),
                    "wam_velocity")
        self._leave()
        return v_out, StepInfo.of(info, self.B)

    def denoise_step(self, k, x, cond, rr=None):
        self._enter()
        info = abi.WamStepInfo()
        self._check(self.lib.wam_denoise_step(self.h, k, _ptr(x), _ptr(cond),
                                              C.byref(rr) if rr is not None else None, C.byref(info)),
                    "wam_denoise_step")
        self._leave()
        return StepInfo.of(info, self.B)

    def continue_(self, k_from, k_to, x, cond, rr=None, capture_stage=-1, x_capture=None):
        self._enter()
        n = max(k_to - k_from, 1)
        infos = (abi.WamStepInfo * n)()
        self._check(self.lib.wam_continue(self.h, k_from, k_to, _ptr(x), _ptr(cond),
                                          C.byref(rr) if rr is not None else None, capture_stage,
                                          _ptr(x_capture), infos), "wam_continue")
        self._leave()
        return [StepInfo.of(infos[i], self.B) for i in range(k_to - k_from)]

    def hidden(self, k, x, cond, n_layers, h_out=None):
        self._enter()
        if h_out is None:
            T = self.cfg.Nv + self.cfg.Na + self.cfg.No
            h_out = torch.empty((self.B, T, self.cfg.D), dtype=torch.float32, device=self.device)
        self._check(self.lib.wam_hidden(self.h, k, _ptr(x), _ptr(cond), n_layers, _ptr(h_out)), "wam_hidden")
        self._leave()
        return h_out

    def remap(self, x_bar, x_r, sigma_r, sigma_b0, shift_action, shift_video, noise, x_out=None):
        self._enter()
        x_out = self.new_traj() if x_out is None else x_out
        a = abi.WamRemapArgs(x_bar=_ptr(x_bar), x_r=_ptr(x_r), sigma_r=sigma_r, sigma_b0=sigma_b0,
                           shift_action=shift_action, shift_video=shift_video, noise=_ptr(noise), x_out=_ptr(x_out))
        self._check(self.lib.wam_adapt_state(self.h, abi.WAM_ADAPT_REMAP, C.byref(a)), "wam_adapt_state(REMAP)")
        self._leave()
        return x_out

    def rebind(self, cond):
        """Observation Rebinding's rebinding step (WAM_ADAPT_REBIND): the retained
        state continues under cond; cond=None in later step calls means it."""
        self._enter()
        a = abi.WamRebindArgs(cond=_ptr(cond))
        self._check(self.lib.wam_adapt_state(self.h, abi.WAM_ADAPT_REBIND, C.byref(a)), "wam_adapt_state(REBIND)")

    def reset_layer_state(self):
        self._check(self.lib.wam_adapt_state(self.h, abi.WAM_ADAPT_RESET_LAYER, None), "RESET_LAYER")

    def reset_all(self):
        self._check(self.lib.wam_adapt_state(self.h, abi.WAM_ADAPT_RESET_ALL, None), "RESET_ALL")

    def set_replan_state(self, x_bar, x_r, kappa):
        self._enter()
        a = abi.WamReplanStateArgs(x_bar=_ptr(x_bar), x_r=_ptr(x_r), kappa=kappa)
        self._check(self.lib.wam_adapt_state(self.h, abi.WAM_ADAPT_SET_REPLAN, C.byref(a)), "SET_REPLAN")

    def get_replan_state(self):
        self._enter()
        xb, xr = self.new_traj(), self.new_traj()
        kappa = C.c_int32()
        self._check(self.lib.wam_get_replan_state(self.h, _ptr(xb), _ptr(xr), C.byref(kappa)),
                    "wam_get_replan_state")
        self._leave()
        return xb, xr, kappa.value

    def consistency_score(self, u_hat, u, delta, weight):
        self._enter()
        n = len(u_hat)
        uh = (C.c_void_p * n)(*[_ptr(t).value for t in u_hat])
        uu = (C.c_void_p * n)(*[_ptr(t).value for t in u])
        cnt = (C.c_int64 * n)(*[t.numel() for t in u])
        dl = (C.c_double * n)(*delta)
        wt = (C.c_double * n)(*weight)
        S = C.c_double()
        self._check(self.lib.wam_consistency_score(self.h, n, uh, uu, cnt, dl, wt, C.byref(S)),
                    "wam_consistency_score")
        self._leave()
        return S.value

    def pack_condition(self, obs, n_obs, c_obs, ctx, n_ctx, c_ctx, ctx_stride, out):
        """out [B][No][Co] = obs tokens then ctx tokens, zero-padded (wam_pack_condition)."""
        self._enter()
        self._check(self.lib.wam_pack_condition(self.h, _ptr(obs), n_obs, c_obs, _ptr(ctx), n_ctx, c_ctx,
                                                ctx_stride, _ptr(out)), "wam_pack_condition")
        self._leave()
        return out

    def replan_args(self, cond_real, x_out, noise_remap, *, cond_pred=None, u_hat=(), u=(), delta=(), weight=(),
                    noise_first=None, rr=None, b0=0, r=0, shift_action=0, shift_video=0, k1=0, tau=0.5,
                    kappa_max=3, tr_enabled=True, or_enabled=True, rr_first=True, rr_prefix=True,
                    rr_refresh=True):
        """The wam_replan_args struct (device buffers referenced, not copied)."""
        a = abi.WamReplanArgs()
        a.cond_real = _ptr(cond_real)
        a.cond_pred = _ptr(cond_pred)
        a.n_components = len(u)
        for m in range(len(u)):
            a.u_hat[m] = _ptr(u_hat[m]).value
            a.u[m] = _ptr(u[m]).value
            a.n[m] = u[m].numel()
            a.delta[m] = delta[m]
            a.weight[m] = weight[m]
        a.noise_first = _ptr(noise_first)
        a.noise_remap = _ptr(noise_remap)
        a.x_out = _ptr(x_out)
        a.rr = rr if rr is not None else rr_profile()
        a.b0, a.r, a.shift_action, a.shift_video, a.k1 = b0, r, shift_action, shift_video, k1
        a.tau, a.kappa_max = tau, kappa_max
        a.tr_enabled, a.or_enabled = int(tr_enabled), int(or_enabled)
        a.rr_first, a.rr_prefix, a.rr_refresh = int(rr_first), int(rr_prefix), int(rr_refresh)
        return a

    def replan(self, cond_real, x_out, noise_remap, **kw):
        self._enter()
        a = self.replan_args(cond_real, x_out, noise_remap, **kw)
        info = abi.WamReplanInfo()
        self._check(self.lib.wam_replan(self.h, C.byref(a), C.byref(info)), "wam_replan")
        self._leave()
        return info

    def replan_begin(self, args):
        """Remap and enqueue the anticipatory prefix (args from replan_args)."""
        self._enter()
        self._check(self.lib.wam_replan_begin(self.h, C.byref(args)), "wam_replan_begin")

    def replan_end(self, args):
        self._enter()
        info = abi.WamReplanInfo()
        self._check(self.lib.wam_replan_end(self.h, C.byref(args), C.byref(info)), "wam_replan_end")
        self._leave()
        return info

    def set_option(self, option, value):
        self._check(self.lib.wam_set_option(self.h, option, int(value)), "wam_set_option")

    def sync(self):
        self._check(self.lib.wam_sync(self.h), "wam_sync")

    def profile_enable(self, kc, enable=True, max_launches=4096):
        self._check(self.lib.wam_profile_enable(self.h, kc, int(enable), max_launches), "wam_profile_enable")

    def profile_read(self, kc):
        t, n, w = C.c_double(), C.c_int64(), C.c_double()
        self._check(self.lib.wam_profile_read(self.h, kc, C.byref(t), C.byref(n), C.byref(w)), "wam_profile_read")
        return t.value, n.value, w.value


class IdmPair:
    """Independently executed video and action models (Sec. 3.3): per control
    step the video model's replan under the observation, then the action
    model's under the observation followed by the video model's new latent
    (packed on the device by wam_pack_condition).  Each model keeps its own
    replan state, schedule, RR decision and graphs."""

    def __init__(self, video: WamModel, action: WamModel, n_obs: int, c_obs: int):
        cv, ca = video.cfg, action.cfg
        if cv.Na != 0 or ca.Nv != 0 or ca.No != n_obs + cv.Nv or ca.Co < max(c_obs, cv.Cv):
            raise WamError("action condition must hold the observation and the video latent tokens")
        self.video, self.action = video, action
        self.n_obs, self.c_obs = n_obs, c_obs
        self.cond_action = torch.zeros((ca.B, ca.No, ca.Co), dtype=torch.float32, device=action.device)

    def replan(self, obs_real, x_video, x_action, noise_remap_video, noise_remap_action, video_kw=None,
               action_kw=None):
        """One control step; returns (video info, action info)."""
        iv = self.video.replan(obs_real, x_video, noise_remap_video, **(video_kw or {}))
        cv = self.video.cfg
        self.action.pack_condition(obs_real, self.n_obs, self.c_obs, x_video, cv.Nv, cv.Cv, self.video.traj,
                                   self.cond_action)
        ia = self.action.replan(self.cond_action, x_action, noise_remap_action, **(action_kw or {}))
        return iv, ia


def remap_noalloc(cfg: abi.WamConfig, x_bar, x_r, sigma_r, sigma_b0, shift_action, shift_video, noise, x_out,
                  stream: torch.cuda.Stream | None = None):
    """Trajectory Remapping without a handle or workspace (wam_remap_noalloc);
    enqueued on stream (default: torch's current stream on x_out's device)."""
    lib = abi.lib()
    s = stream if stream is not None else torch.cuda.current_stream(x_out.device)
    a = abi.WamRemapArgs(x_bar=_ptr(x_bar), x_r=_ptr(x_r), sigma_r=sigma_r, sigma_b0=sigma_b0,
                         shift_action=shift_action, shift_video=shift_video, noise=_ptr(noise), x_out=_ptr(x_out))
    rc = lib.wam_remap_noalloc(C.byref(cfg), C.byref(a), C.c_void_p(s.cuda_stream))
    if rc != abi.WAM_OK:
        raise WamError(f"wam_remap_noalloc: {lib.wam_status_string(rc).decode()}: "
                       f"{lib.wam_noalloc_last_error().decode()}")
    return x_out


def probe_mfma_bf16(shape: int = 0, n_blocks: int = 1024, iters: int = 20000, device="cuda:0"):
    """Achievable bf16 MFMA rate (wam_probe_mfma_bf16): returns (TFLOP/s, ms)."""
    lib = abi.lib()
    sink = torch.empty(n_blocks * 256, dtype=torch.float32, device=device)
    stream = C.c_void_p(torch.cuda.current_stream(sink.device).cuda_stream)
    tf, ms = C.c_double(), C.c_double()
    rc = lib.wam_probe_mfma_bf16(stream, shape, n_blocks, iters, _ptr(sink), C.byref(tf), C.byref(ms))
    if rc != abi.WAM_OK:
        raise WamError(f"wam_probe_mfma_bf16: {lib.wam_status_string(rc).decode()}")
    return tf.value, ms.value


def probe_copy(nbytes: int = 1 << 30, reps: int = 5, device="cuda:0"):
    """Achievable streaming copy rate (wam_probe_copy): returns (GB/s counting
    read + write bytes, ms per copy)."""
    lib = abi.lib()
    n = nbytes // 4
    src = torch.ones(n, dtype=torch.float32, device=device)
    dst = torch.empty_like(src)
    stream = C.c_void_p(torch.cuda.current_stream(src.device).cuda_stream)
    gbs, ms = C.c_double(), C.c_double()
    rc = lib.wam_probe_copy(stream, _ptr(src), _ptr(dst), n * 4, reps, C.byref(gbs), C.byref(ms))
    if rc != abi.WAM_OK:
        raise WamError(f"wam_probe_copy: {lib.wam_status_string(rc).decode()}")
    return gbs.value, ms.value
