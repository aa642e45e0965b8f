"""ctypes binding of the f3c C ABI (include/f3c.h).

Argument marshalling only: every call forwards to libf3c.so, which runs every
step of the cached sampler in HIP kernels. Device memory and streams come from
PyTorch (``torch.empty(..., device="cuda")`` buffers and the current stream);
nothing here computes any part of the method.

If the library has not been built, ``lib()`` raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Dict, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "lib", "libf3c.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "f3c.h")

F3C_OK, F3C_EINVAL, F3C_ENOMEM, F3C_EHIP, F3C_ESTATE = 0, -1, -2, -3, -4
F3C_F32, F3C_BF16 = 0, 1
F3C_STATE_GUIDED = 1
PROF_CLASSES = ["select", "embed", "mod", "ln", "gemm_qkv", "attn_self", "gemm_o", "gemm_q", "attn_cross",
                "gemm_co", "gemm_fc1", "gemm_fc2", "final", "euler", "cond"]

c_int, c_i64, c_f, c_d, c_sz, c_p = (ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double,
                                     ctypes.c_size_t, ctypes.c_void_p)
P_i32 = ctypes.POINTER(ctypes.c_int32)
P_f = ctypes.POINTER(ctypes.c_float)
P_d = ctypes.POINTER(ctypes.c_double)


class F3CError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"f3c error {code}: {msg}")
        self.code = code


class ModelCfg(ctypes.Structure):
    _fields_ = [(n, c_int) for n in ("grid", "in_ch", "width", "depth", "heads", "mlp_ratio", "cond_tokens",
                                     "cond_width", "dtype")]


_SIGS = {
    "f3c_last_error": (ctypes.c_char_p, []),
    "f3c_version": (c_int, []),
    "f3c_model_create": (c_int, [ctypes.POINTER(ModelCfg), ctypes.POINTER(c_p)]),
    "f3c_model_destroy": (None, [c_p]),
    "f3c_weight_count": (c_int, [c_p, P_i32]),
    "f3c_weight_info": (c_int, [c_p, c_int, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(c_i64)]),
    "f3c_model_weights_bytes": (c_int, [c_p, ctypes.POINTER(c_sz)]),
    "f3c_model_load_weights": (c_int, [c_p, c_p, c_sz, ctypes.POINTER(P_f), c_int]),
    "f3c_forward_flops": (c_d, [ctypes.POINTER(ModelCfg), c_int, c_int]),
    "f3c_state_bytes": (c_int, [c_p, c_int, ctypes.POINTER(c_sz)]),
    "f3c_state_create": (c_int, [c_p, c_int, c_p, c_sz, c_p, ctypes.POINTER(c_p)]),
    "f3c_state_bytes_ex": (c_int, [c_p, c_int, ctypes.c_uint32, ctypes.POINTER(c_sz)]),
    "f3c_state_create_ex": (c_int, [c_p, c_int, ctypes.c_uint32, c_p, c_sz, c_p, ctypes.POINTER(c_p)]),
    "f3c_set_uncond": (c_int, [c_p, c_p, c_p]),
    "f3c_plan_bytes": (c_int, [c_p, c_int, ctypes.POINTER(c_sz)]),
    "f3c_state_plan_times": (c_int, [c_p, P_d, c_int, c_p, c_sz, c_p]),
    "f3c_guided_step": (c_int, [c_p, c_p, c_d, c_d, P_i32, c_d, c_p]),
    "f3c_guidance_active": (c_int, [c_d, c_d, c_d]),
    "f3c_state_trace_blocks": (c_int, [c_p, c_p, c_sz]),
    "f3c_state_trace_sublayers": (c_int, [c_p, c_p, c_sz]),
    "f3c_debug_force_active": (c_int, [c_p, c_p]),
    "f3c_state_destroy": (None, [c_p]),
    "f3c_state_reset": (c_int, [c_p, c_p]),
    "f3c_state_set_omega": (c_int, [c_p, c_f]),
    "f3c_set_cond": (c_int, [c_p, c_p, c_p]),
    "f3c_full_step": (c_int, [c_p, c_p, c_d, c_d, c_p]),
    "f3c_cached_step": (c_int, [c_p, c_p, c_d, c_d, P_i32, c_p]),
    "f3c_state_views": (c_int, [c_p] + [ctypes.POINTER(c_p)] * 7 + [P_i32]),
    "f3c_state_record_scores": (c_int, [c_p, c_int]),
    "f3c_state_export": (c_int, [c_p, P_f, c_sz, c_p]),
    "f3c_state_import": (c_int, [c_p, P_f, c_sz, c_p]),
    "f3c_profile_enable": (c_int, [c_p, ctypes.c_uint32]),
    "f3c_profile_read": (c_int, [c_p, c_int, ctypes.POINTER(c_i64), P_d, P_d, P_d]),
    "f3c_profile_reset": (c_int, [c_p]),
    "f3c_op_select": (c_int, [c_int, c_int, c_p, c_p, c_f, P_i32, c_p, c_p, c_p, c_p, c_sz, c_p]),
    "f3c_op_select_workspace_bytes": (c_int, [c_int, c_int, ctypes.POINTER(c_sz)]),
    "f3c_op_select_noalloc": (c_int, [c_int, c_int, c_p, c_p, c_f, P_i32, c_p, c_p, c_p, c_p]),
    "f3c_op_select_scores": (c_int, [c_int, c_int, c_p, P_i32, c_p, c_p, c_p]),
    "f3c_op_gemm": (c_int, [c_int, c_int, c_int, c_int, c_int, c_p, c_int, c_p, c_int, c_p, c_p, c_p, c_int, c_p,
                            c_int, c_p]),
    "f3c_op_attention": (c_int, [c_int, c_int, c_int, c_int, P_i32, P_i32, c_p, c_int, c_p, c_int, c_p, c_int, c_p,
                                 c_int, c_p, c_sz, c_int, c_p]),
    "f3c_op_ln_mod": (c_int, [c_int, c_int, c_int, c_p, c_p, c_p, c_p, c_p]),
    "f3c_op_modulation": (c_int, [c_p, c_d, c_p, c_p, c_p]),
    "f3c_op_embed": (c_int, [c_p, c_int, c_p, c_p, P_i32, c_p, c_p]),
    "f3c_op_final": (c_int, [c_p, c_int, c_p, c_p, c_p]),
    "f3c_op_euler": (c_int, [c_int, c_int, c_p, c_p, c_p, c_p, P_i32, c_d, c_d, c_p, c_p]),
    "f3c_op_pack_occupancy": (c_int, [c_int, c_i64, c_p, c_p, c_p]),
    "f3c_op_dynamic_voxels": (c_int, [c_int, c_i64, c_p, c_p, c_p, c_p]),
    "f3c_time_grid": (c_int, [c_int, c_d, P_d]),
    "f3c_ceil_ratio": (c_int, [c_int, c_d]),
    "f3c_pcsc_quota": (c_int, [c_int, c_int, c_d, c_d, c_int, c_d]),
    "f3c_phase_quota": (c_int, [c_int, c_int, c_int, c_int, c_d, c_d, c_d, c_int]),
    "f3c_tau_forces_full": (c_int, [c_int, c_int, c_int]),
    "f3c_schedule_plan": (c_int, [ctypes.c_void_p, c_d, P_i32]),
}

_lib: Optional[ctypes.CDLL] = None


def lib() -> ctypes.CDLL:
    """Load libf3c.so (built in-tree by build.py); raise if it is missing."""
    global _lib
    if _lib is None:
        # PyTorch ships its own HIP runtime (same soname). Importing it first makes
        # libf3c.so bind to that runtime, so streams and allocations are shared
        # by one runtime instance in the process.
        import torch  # noqa: F401
        if not os.path.exists(LIB_PATH):
            raise F3CError(F3C_ESTATE, f"{LIB_PATH} not built; run paper_2511_22533_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def header_symbols() -> list:
    """Function names declared in include/f3c.h."""
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(f3c_[a-z_0-9]+)\s*\(", text)))


def check(rc: int) -> None:
    if rc != F3C_OK:
        raise F3CError(rc, lib().f3c_last_error().decode())


def _i32(a: Sequence[int]):
    arr = (ctypes.c_int32 * len(a))(*[int(x) for x in a])
    return arr


def model_cfg(cfg) -> ModelCfg:
    """ModelCfg from a synth.ModelConfig."""
    return ModelCfg(cfg.grid, cfg.in_ch, cfg.width, cfg.depth, cfg.heads, cfg.mlp_ratio, cfg.cond_tokens,
                    cfg.cond_width, F3C_BF16 if cfg.dtype == "bf16" else F3C_F32)


def _stream(stream) -> int:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return int(stream)


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


# ---------------------------------------------------------------- host schedules

def time_grid(steps: int, eta: float) -> np.ndarray:
    out = (ctypes.c_double * (steps + 1))()
    check(lib().f3c_time_grid(steps, eta, out))
    return np.array(out[:], dtype=np.float64)


def ceil_ratio(steps: int, rho: float) -> int:
    return int(lib().f3c_ceil_ratio(steps, rho))


def pcsc_quota(k, n_tokens, sigma, mu, k_anchor, gamma_up) -> int:
    return int(lib().f3c_pcsc_quota(k, n_tokens, sigma, mu, k_anchor, gamma_up))


def phase_quota(k, steps, n_tokens, n_cache_phase2, rho_a=0.2, rho_off=0.75, xi=0.7, f_corr=3) -> int:
    return int(lib().f3c_phase_quota(k, steps, n_tokens, n_cache_phase2, rho_a, rho_off, xi, f_corr))


TAU_CYCLE, TAU_LITERAL = 0, 1


class ScheduleCfg(ctypes.Structure):
    _fields_ = [("steps", c_int), ("n_tokens", c_int), ("rho_a", c_d), ("rho_off", c_d), ("xi", c_d),
                ("f_corr", c_int), ("mu", c_d), ("gamma_up", c_d), ("tau", c_int), ("tau_reading", c_int)]


def guidance_active(t: float, lo: float = 0.5, hi: float = 1.0) -> bool:
    return bool(lib().f3c_guidance_active(t, lo, hi))


def tau_forces_full(consecutive: int, tau: int, reading: int = TAU_CYCLE) -> bool:
    return bool(lib().f3c_tau_forces_full(consecutive, tau, reading))


def schedule_plan(steps: int, n_tokens: int, sigma: float, mu: float = -0.07, gamma_up: float = 1.0,
                  rho_a: float = 0.2, rho_off: float = 0.75, xi: float = 0.7, f_corr: int = 3, tau: int = 0,
                  reading: int = TAU_CYCLE) -> np.ndarray:
    c = ScheduleCfg(steps, n_tokens, rho_a, rho_off, xi, f_corr, mu, gamma_up, tau, reading)
    out = (ctypes.c_int32 * steps)()
    check(lib().f3c_schedule_plan(ctypes.byref(c), sigma, out))
    return np.array(out[:], dtype=np.int32)


def forward_flops(cfg, n_tok: int, batch: int = 1) -> float:
    c = model_cfg(cfg)
    return float(lib().f3c_forward_flops(ctypes.byref(c), n_tok, batch))


# ---------------------------------------------------------------- model / state

class Model:
    """A model handle plus its torch-allocated weight buffer."""

    def __init__(self, cfg):
        self.cfg = cfg
        self.c = model_cfg(cfg)
        h = c_p()
        check(lib().f3c_model_create(ctypes.byref(self.c), ctypes.byref(h)))
        self.h = h
        self.wbuf = None

    def weight_names(self):
        n = c_int()
        check(lib().f3c_weight_count(self.h, ctypes.byref(n)))
        out = []
        for i in range(n.value):
            name, numel = ctypes.c_char_p(), c_i64()
            check(lib().f3c_weight_info(self.h, i, ctypes.byref(name), ctypes.byref(numel)))
            out.append((name.value.decode(), numel.value))
        return out

    def weights_bytes(self) -> int:
        b = c_sz()
        check(lib().f3c_model_weights_bytes(self.h, ctypes.byref(b)))
        return b.value

    def load(self, weights: Dict[str, np.ndarray]):
        import torch
        names = self.weight_names()
        arrs = []
        for name, numel in names:
            a = np.ascontiguousarray(weights[name], dtype=np.float32).reshape(-1)
            if a.size != numel:
                raise F3CError(F3C_EINVAL, f"{name}: expected {numel} values, got {a.size}")
            arrs.append(a)
        self.wbuf = torch.empty(self.weights_bytes(), dtype=torch.uint8, device="cuda")
        ptrs = (P_f * len(arrs))(*[a.ctypes.data_as(P_f) for a in arrs])
        check(lib().f3c_model_load_weights(self.h, self.wbuf.data_ptr(), self.wbuf.numel(), ptrs, len(arrs)))
        return self

    def modulation(self, t: float, stream=None):
        import torch
        mod = torch.empty(self.cfg.depth * 6 * self.cfg.width, dtype=torch.float32, device="cuda")
        scratch = torch.empty(2 * self.cfg.width, dtype=torch.float32, device="cuda")
        check(lib().f3c_op_modulation(self.h, t, mod.data_ptr(), scratch.data_ptr(), _stream(stream)))
        return mod.view(self.cfg.depth, 6, self.cfg.width)

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.f3c_model_destroy(self.h)
            self.h = None


class State:
    """A sampler state (velocity caches, activations, condition K/V) of one model.

    guided=True sizes it for guided steps (two transformer passes per sample)."""

    def __init__(self, model: Model, batch: int, stream=None, guided: bool = False):
        import torch
        self.model, self.batch, self.guided = model, batch, guided
        flags = F3C_STATE_GUIDED if guided else 0
        b = c_sz()
        check(lib().f3c_state_bytes_ex(model.h, batch, flags, ctypes.byref(b)))
        self.buf = torch.empty(b.value, dtype=torch.uint8, device="cuda")
        h = c_p()
        check(lib().f3c_state_create_ex(model.h, batch, flags, self.buf.data_ptr(), self.buf.numel(),
                                        _stream(stream), ctypes.byref(h)))
        self.h = h
        self.last_guided = False
        self.plan_buf = None

    def reset(self, stream=None):
        check(lib().f3c_state_reset(self.h, _stream(stream)))

    def set_omega(self, omega: float):
        check(lib().f3c_state_set_omega(self.h, omega))

    def set_cond(self, cond, stream=None):
        check(lib().f3c_set_cond(self.h, cond.data_ptr(), _stream(stream)))

    def set_uncond(self, uncond, stream=None):
        check(lib().f3c_set_uncond(self.h, uncond.data_ptr(), _stream(stream)))

    def plan_times(self, times: Sequence[float], stream=None):
        """Plan the timestep modulation of these times (normally the trajectory's
        time grid): later steps at exactly one of them read it instead of
        recomputing it. An empty sequence clears the plan. The plan's device
        buffer belongs to this object and is reused while it is large enough."""
        import torch
        t = [float(v) for v in times]
        if not t:
            check(lib().f3c_state_plan_times(self.h, None, 0, None, 0, _stream(stream)))
            return
        b = c_sz()
        check(lib().f3c_plan_bytes(self.model.h, len(t), ctypes.byref(b)))
        if self.plan_buf is None or self.plan_buf.numel() < b.value:
            self.plan_buf = torch.empty(b.value, dtype=torch.uint8, device="cuda")
        check(lib().f3c_state_plan_times(self.h, (c_d * len(t))(*t), len(t), self.plan_buf.data_ptr(),
                                         self.plan_buf.numel(), _stream(stream)))

    def full_step(self, x, t: float, t_next: float, stream=None):
        check(lib().f3c_full_step(self.h, x.data_ptr(), t, t_next, _stream(stream)))
        self.last_guided = False

    def cached_step(self, x, t: float, t_next: float, n_cache: Sequence[int], stream=None):
        check(lib().f3c_cached_step(self.h, x.data_ptr(), t, t_next, _i32(n_cache), _stream(stream)))
        self.last_guided = False

    def guided_step(self, x, t: float, t_next: float, n_cache: Optional[Sequence[int]], w: float, stream=None):
        """Guided step; n_cache None runs every token."""
        check(lib().f3c_guided_step(self.h, x.data_ptr(), t, t_next, None if n_cache is None else _i32(n_cache), w,
                                    _stream(stream)))
        self.last_guided = True

    def trace_blocks(self, buf=None):
        """Debug: copy the residual stream after the embedding and each block into buf (f32 device tensor)."""
        check(lib().f3c_state_trace_blocks(self.h, _ptr(buf), buf.numel() * 4 if buf is not None else 0))

    def trace_sublayers(self, buf=None):
        """Debug: write each block's pre-gate sublayer outputs into buf (f32 device tensor [L][3][rows][width])."""
        check(lib().f3c_state_trace_sublayers(self.h, _ptr(buf), buf.numel() * 4 if buf is not None else 0))

    def force_active(self, idx_active=None):
        """Debug: the next step uses these active sets (int32 device tensor, per sample ascending,
        concatenated) instead of its own selection; None disarms."""
        check(lib().f3c_debug_force_active(self.h, _ptr(idx_active)))
        self._forced = idx_active          # kept alive until the step has run

    def record_scores(self, on: bool):
        check(lib().f3c_state_record_scores(self.h, int(on)))

    def views(self):
        """Device pointers of the caches/selection and the last step's active offsets."""
        ps = [c_p() for _ in range(7)]
        off = (ctypes.c_int32 * (self.batch + 1))()
        check(lib().f3c_state_views(self.h, *[ctypes.byref(p) for p in ps], off))
        keys = ["v_cache", "v_prev", "idx_active", "pos", "v_act", "mod", "score"]
        out = {k: p.value for k, p in zip(keys, ps)}
        out["act_off"] = list(off)
        return out

    def tensors(self):
        """Zero-copy torch views of the state's device buffers (caches, selection, v_act, mod, score)."""
        import torch
        v = self.views()
        cfg, B = self.model.cfg, self.batch
        N = cfg.tokens
        rows = v["act_off"][-1]

        def view(ptr, n, dtype, shape):
            if ptr is None:
                return None
            nbytes = n * torch.empty((), dtype=dtype).element_size()
            for owner in (self.buf, self.plan_buf):   # the state's buffer, or the modulation plan's
                if owner is not None and owner.data_ptr() <= ptr and ptr + nbytes <= owner.data_ptr() + owner.numel():
                    off = ptr - owner.data_ptr()
                    return owner[off:off + nbytes].view(dtype).view(shape)
            raise F3CError(F3C_EINVAL, "view outside the state's buffers")

        return {
            "v_cache": view(v["v_cache"], B * N * 8, torch.float32, (B, N, 8)),
            "v_prev": view(v["v_prev"], B * N * 8, torch.float32, (B, N, 8)),
            "idx_active": view(v["idx_active"], rows, torch.int32, (rows,)),
            "pos": view(v["pos"], B * N, torch.int32, (B, N)),
            # a guided step leaves the conditional rows followed by the unconditional ones
            "v_act": view(v["v_act"], (2 if self.last_guided else 1) * rows * 8, torch.float32,
                          ((2 if self.last_guided else 1) * rows, 8)),
            "mod": view(v["mod"], cfg.depth * 6 * cfg.width, torch.float32, (cfg.depth, 6, cfg.width)),
            "score": view(v["score"], B * N, torch.float32, (B, N)),
            "act_off": v["act_off"],
        }

    def export(self, stream=None) -> np.ndarray:
        n = 2 * self.batch * self.model.cfg.tokens * 8
        host = np.empty(n, np.float32)
        check(lib().f3c_state_export(self.h, host.ctypes.data_as(P_f), n, _stream(stream)))
        return host

    def import_(self, host: np.ndarray, stream=None):
        host = np.ascontiguousarray(host, dtype=np.float32)
        check(lib().f3c_state_import(self.h, host.ctypes.data_as(P_f), host.size, _stream(stream)))

    def profile(self, classes=None):
        """Record HIP events around launches of the named kernel classes (all if True, none if falsy)."""
        if classes is True:
            mask = (1 << len(PROF_CLASSES)) - 1
        elif not classes:
            mask = 0
        else:
            mask = 0
            for c in classes:
                mask |= 1 << PROF_CLASSES.index(c)
        check(lib().f3c_profile_enable(self.h, mask))

    def profile_reset(self):
        check(lib().f3c_profile_reset(self.h))

    def profile_read(self) -> Dict[str, dict]:
        out = {}
        for i, name in enumerate(PROF_CLASSES):
            n, ms, fl, by = c_i64(), c_d(), c_d(), c_d()
            check(lib().f3c_profile_read(self.h, i, ctypes.byref(n), ctypes.byref(ms), ctypes.byref(fl),
                                         ctypes.byref(by)))
            out[name] = {"launches": n.value, "ms": ms.value, "flops": fl.value, "bytes": by.value}
        return out

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.f3c_state_destroy(self.h)
            self.h = None


# ---------------------------------------------------------------- operator calls

def select_workspace_bytes(batch: int, n_tokens: int) -> int:
    b = c_sz()
    check(lib().f3c_op_select_workspace_bytes(batch, n_tokens, ctypes.byref(b)))
    return b.value


def op_select(v_cache, v_prev, omega: float, n_cache: Sequence[int], idx_active, pos, score=None, workspace=None,
              stream=None):
    """workspace: a device uint8 tensor of at least select_workspace_bytes(B, N) (allocated here if None)."""
    import torch
    B, N = v_cache.shape[0], v_cache.shape[1]
    if workspace is None:
        workspace = torch.empty(select_workspace_bytes(B, N), dtype=torch.uint8, device=v_cache.device)
    check(lib().f3c_op_select(B, N, v_cache.data_ptr(), v_prev.data_ptr(), omega, _i32(n_cache),
                              idx_active.data_ptr(), pos.data_ptr(), _ptr(score), workspace.data_ptr(),
                              workspace.numel() * workspace.element_size(), _stream(stream)))


def op_select_noalloc(v_cache, v_prev, omega: float, n_cache: Sequence[int], idx_active, pos, score=None,
                      stream=None):
    """op_select with the library's static scratch (allocates nothing)."""
    B, N = v_cache.shape[0], v_cache.shape[1]
    check(lib().f3c_op_select_noalloc(B, N, v_cache.data_ptr(), v_prev.data_ptr(), omega, _i32(n_cache),
                                      idx_active.data_ptr(), pos.data_ptr(), _ptr(score), _stream(stream)))


def op_select_scores(scores, n_cache: Sequence[int], idx_active, pos, stream=None):
    """The selection alone from given float32 scores [B][N] (device)."""
    B, N = scores.shape[0], scores.shape[1]
    check(lib().f3c_op_select_scores(B, N, scores.data_ptr(), _i32(n_cache), idx_active.data_ptr(), pos.data_ptr(),
                                     _stream(stream)))


def op_gemm(dtype: int, epilogue: int, A, W, bias, out=None, resid=None, gate=None, stream=None):
    M, K = A.shape
    N = W.shape[0]
    check(lib().f3c_op_gemm(dtype, epilogue, M, N, K, A.data_ptr(), A.stride(0), W.data_ptr(), W.stride(0),
                            bias.data_ptr(), _ptr(gate), _ptr(out), out.stride(0) if out is not None else 0,
                            _ptr(resid), resid.stride(0) if resid is not None else 0, _stream(stream)))


def attention_q_scale(head_dim: int) -> float:
    """log2(e) / sqrt(head_dim): the factor of pre-scaled queries (q_prescaled)."""
    import math
    return float(np.float32(1.4426950408889634) / np.float32(math.sqrt(head_dim)))


def op_attention(dtype: int, heads: int, head_dim: int, q_off, k_off, q, k, v, o, workspace=None, stream=None,
                 q_prescaled: bool = False):
    B = len(q_off) - 1
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    check(lib().f3c_op_attention(dtype, heads, head_dim, B, _i32(q_off), _i32(k_off), q.data_ptr(), q.stride(0),
                                 k.data_ptr(), k.stride(0), v.data_ptr(), v.stride(0), o.data_ptr(), o.stride(0),
                                 _ptr(workspace), ws_bytes, int(q_prescaled), _stream(stream)))


def op_embed(model: "Model", x, act_off, h, idx_active=None, stream=None):
    B = len(act_off) - 1
    check(lib().f3c_op_embed(model.h, B, x.data_ptr(), _ptr(idx_active), _i32(act_off), h.data_ptr(),
                             _stream(stream)))


def op_final(model: "Model", h, v_act, stream=None):
    check(lib().f3c_op_final(model.h, h.shape[0], h.data_ptr(), v_act.data_ptr(), _stream(stream)))


def op_euler(x, v_cache, v_act, pos, act_off, t: float, t_next: float, v_new, stream=None):
    B, N = x.shape[0], x.shape[1]
    check(lib().f3c_op_euler(B, N, x.data_ptr(), v_cache.data_ptr(), _ptr(v_act), _ptr(pos), _i32(act_off),
                             float(t), float(t_next), v_new.data_ptr(), _stream(stream)))


def op_pack_occupancy(logits, bits, stream=None):
    """logits f32 [B][n_voxels] -> bits int32/uint32 [B][ceil(n_voxels / 32)] (device tensors)."""
    B, n = logits.shape[0], logits[0].numel()
    if not (logits.is_contiguous() and bits.is_contiguous() and bits.numel() == B * ((n + 31) // 32)):
        raise ValueError("logits [B][n] and bits [B][ceil(n/32)] must be contiguous")
    check(lib().f3c_op_pack_occupancy(B, n, logits.data_ptr(), bits.data_ptr(), _stream(stream)))


def op_dynamic_voxels(occ_next, occ_prev, counts, stream=None):
    """Packed grids [B][n_words] (device) -> counts int64 [B] (device), Eq. (1)."""
    B, n_words = occ_next.shape[0], occ_next[0].numel()
    if not (occ_next.is_contiguous() and occ_prev.is_contiguous() and occ_prev.shape == occ_next.shape
            and counts.numel() == B):
        raise ValueError("occ_next, occ_prev [B][n_words] contiguous and counts [B] expected")
    check(lib().f3c_op_dynamic_voxels(B, n_words, occ_next.data_ptr(), occ_prev.data_ptr(), counts.data_ptr(),
                                      _stream(stream)))


def op_ln_mod(dtype: int, h, out, shift=None, scale=None, stream=None):
    rows, d = h.shape
    check(lib().f3c_op_ln_mod(dtype, rows, d, h.data_ptr(), _ptr(shift), _ptr(scale), out.data_ptr(),
                              _stream(stream)))
