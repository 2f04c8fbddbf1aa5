"""ctypes binding of libdllm.so (the C ABI in include/dllm.h).

Argument marshalling only: every step of the decode runs in the library's HIP
kernels.  PyTorch supplies device memory and the stream.  Importing this
module does not load the library; ``lib()`` does, and raises if the library
has not been built (python -m paper_2608_22646_amd.build).
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdllm.so")

DLLM_F32, DLLM_BF16 = 0, 1
F_BLOCK_SCHED, F_POS, F_BUDGET, F_GRIND, F_FIXED = 1, 2, 4, 8, 16
R_MASKED, R_THRESH, R_BUDGET, R_GRIND, R_FLUSH, R_FIXED = 0, 1, 2, 3, 4, 5
PROF_QKV, PROF_ATTN, PROF_HEAD, PROF_COMMIT, PROF_NORM, PROF_GATEUP, PROF_OPROJ, PROF_DOWN = range(8)

_c = ctypes
_i32, _u32, _f32, _f64, _vp, _sz = _c.c_int32, _c.c_uint32, _c.c_float, _c.c_double, _c.c_void_p, _c.c_size_t


class ModelCfg(_c.Structure):
    _fields_ = [("n_layers", _i32), ("d_model", _i32), ("n_heads", _i32), ("n_kv_heads", _i32),
                ("head_dim", _i32), ("d_ff", _i32), ("vocab", _i32), ("mask_id", _i32),
                ("rms_eps", _f32), ("rope_base", _f64), ("dtype", _i32)]


class CaiParams(_c.Structure):
    _fields_ = [("block_len", _i32), ("steps_per_block", _i32),
                ("theta_s", _f64), ("theta_e", _f64), ("theta_e_step", _f64), ("theta_e_floor", _f64),
                ("warmup", _f64), ("pos_edge", _i32 * 3), ("pos_factor", _f64 * 4),
                ("clip_lo", _f64), ("clip_hi", _f64), ("s_easy", _f32), ("s_hard", _f32),
                ("p_easy", _i32), ("p_hard", _i32), ("budget_easy", _i32), ("budget_mid", _i32),
                ("budget_hard", _i32), ("eta_bar", _f64), ("patience", _i32), ("theta_fb", _f32),
                ("flags", _u32)]


class State(_c.Structure):
    _fields_ = [("x", _vp), ("commit_step", _vp), ("reason", _vp), ("s", _vp), ("budget", _vp),
                ("ell", _vp), ("done", _vp)]


class WsLayout(_c.Structure):
    _fields_ = [(n, _sz) for n in ("total", "h", "a_attn", "q", "k", "vt", "attn", "a_mlp", "u", "hb")]


class DllmError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"dllm error {code}: {msg}")
        self.code = code


_LIB = None

_SIGS = {
    "dllm_last_error": (_c.c_char_p, []),
    "dllm_model_buffer_size": (_i32, [_c.POINTER(ModelCfg), _c.POINTER(_sz)]),
    "dllm_model_create": (_i32, [_c.POINTER(ModelCfg), _c.POINTER(_vp), _i32, _vp, _sz, _vp, _c.POINTER(_vp)]),
    "dllm_model_destroy": (_i32, [_vp]),
    "dllm_model_packed_size": (_i32, [_vp, _c.POINTER(_sz)]),
    "dllm_model_pack_weights": (_i32, [_vp, _vp, _sz, _vp]),
    "dllm_workspace_size": (_i32, [_vp, _i32, _i32, _i32, _c.POINTER(_sz)]),
    "dllm_workspace_layout": (_i32, [_vp, _i32, _i32, _i32, _c.POINTER(WsLayout)]),
    "dllm_embed": (_i32, [_vp, _vp, _i32, _i32, _vp, _sz, _vp]),
    "dllm_layer": (_i32, [_vp, _i32, _i32, _i32, _i32, _vp, _sz, _vp]),
    "dllm_head": (_i32, [_vp, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _sz, _vp]),
    "dllm_forward": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _sz, _vp]),
    "dllm_head_noalloc": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp]),
    "dllm_state_init": (_i32, [_i32, _vp, _i32, _i32, _i32, _c.POINTER(State), _vp]),
    "dllm_commit": (_i32, [_c.POINTER(CaiParams), _c.POINTER(State), _vp, _vp, _i32, _i32, _i32, _i32, _i32,
                           _i32, _vp, _vp]),
    "dllm_step": (_i32, [_vp, _c.POINTER(CaiParams), _c.POINTER(State), _i32, _i32, _i32, _i32, _i32, _vp, _vp,
                         _vp, _vp, _sz, _vp]),
    "dllm_generate": (_i32, [_vp, _c.POINTER(CaiParams), _vp, _i32, _i32, _i32, _c.POINTER(State), _vp, _vp,
                             _vp, _vp, _vp, _sz, _vp]),
    "dllm_kv_cache_size": (_i32, [_vp, _i32, _i32, _c.POINTER(_sz)]),
    "dllm_forward_kv": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _sz, _vp, _sz, _vp]),
    "dllm_embed_rows": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _vp, _sz, _vp]),
    "dllm_layer_kv": (_i32, [_vp, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _sz, _vp, _sz, _vp]),
    "dllm_step_kv": (_i32, [_vp, _c.POINTER(CaiParams), _i32, _c.POINTER(State), _i32, _i32, _i32, _i32, _i32, _vp,
                            _vp, _vp, _vp, _sz, _vp, _sz, _vp]),
    "dllm_generate_kv": (_i32, [_vp, _c.POINTER(CaiParams), _i32, _vp, _i32, _i32, _i32, _c.POINTER(State), _vp,
                                _vp, _vp, _vp, _vp, _sz, _vp, _sz, _vp]),
    "dllm_prof_enable": (_i32, [_vp, _i32]),
    "dllm_prof_read": (_i32, [_vp, _i32, _c.POINTER(_f64), _c.POINTER(_c.c_int64)]),
    "dllm_prof_every": (_i32, [_vp, _i32]),
}


def lib():
    """Load libdllm.so (once).  Raises if it has not been built."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with python -m paper_2608_22646_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _LIB = L
    return _LIB


def check(rc):
    if rc != 0:
        raise DllmError(rc, lib().dllm_last_error().decode())
    return rc


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def device_buffer(nbytes, device="cuda"):
    """A caller-owned, 256-byte aligned uint8 device tensor of nbytes bytes."""
    buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
    off = (-buf.data_ptr()) % 256
    return buf[off:off + nbytes]


# ---------------------------------------------------------------- parameters
@dataclass
class Controller:
    """Controller constants (defaults as printed in the paper, Boxes 3-7)."""
    block_len: int = 32
    steps_per_block: int = 0
    theta_s: float = 0.90
    theta_e: float = 0.70
    theta_e_step: float = 0.10
    theta_e_floor: float = 0.40
    warmup: float = 0.15
    pos_edges: tuple = (16, 32, 48)
    pos_factors: tuple = (0.80, 0.90, 1.05, 1.10)
    clip_lo: float = 0.20
    clip_hi: float = 0.98
    s_easy: float = 0.50
    s_hard: float = 0.25
    p_easy: int = 32
    p_hard: int = 48
    budget_easy: int = 8
    budget_mid: int = 32
    budget_hard: int = 64
    eta_bar: float = 1.5
    patience: int = 4
    theta_fb: float = 0.40
    block_sched: bool = True
    pos_aware: bool = True
    budgets: bool = True
    grinding: bool = True
    fixed: bool = False   # fixed-schedule baseline instead of the confidence rule

    @classmethod
    def gating(cls, on: bool, **kw):
        return cls(budgets=on, grinding=on, **kw)

    @classmethod
    def preset(cls, name: str, **kw):
        """Named controller settings: the method with gating on / off (Section 4.6),
        the component ablation of Section 6 (+APD, +Block, +Budget = the
        per-token controls of Boxes 5-7), fixed-threshold decoding and the
        fixed-schedule baseline.  Keyword arguments override fields."""
        apd_only = dict(block_sched=False, pos_aware=False, budgets=False, grinding=False)
        table = {
            "cai": {},
            "cai_gate_off": dict(budgets=False, grinding=False),
            "apd": apd_only,
            "apd_block": dict(pos_aware=False, budgets=False, grinding=False),
            "apd_block_budget": {},
            "fixed_threshold_0.9": dict(apd_only, theta_s=0.9, theta_e=0.9),
            "fixed_threshold_0.7": dict(apd_only, theta_s=0.7, theta_e=0.7),
            "apd_0.9_to_0.5": dict(apd_only, theta_s=0.9, theta_e=0.5),
            "fixed_schedule": dict(fixed=True),
        }
        if name not in table:
            raise KeyError(f"unknown controller preset {name!r}; known: {sorted(table)}")
        return cls(**dict(table[name], **kw))

    def to_c(self) -> CaiParams:
        p = CaiParams()
        for f in ("block_len", "steps_per_block", "theta_s", "theta_e", "theta_e_step", "theta_e_floor", "warmup",
                  "clip_lo", "clip_hi", "s_easy", "s_hard", "p_easy", "p_hard", "budget_easy", "budget_mid",
                  "budget_hard", "eta_bar", "patience", "theta_fb"):
            setattr(p, f, getattr(self, f))
        p.pos_edge[:] = list(self.pos_edges)
        p.pos_factor[:] = list(self.pos_factors)
        p.flags = ((F_BLOCK_SCHED if self.block_sched else 0) | (F_POS if self.pos_aware else 0)
                   | (F_BUDGET if self.budgets else 0) | (F_GRIND if self.grinding else 0)
                   | (F_FIXED if self.fixed else 0))
        return p

    @property
    def T(self):
        return self.steps_per_block or self.block_len


def model_cfg(cfg) -> ModelCfg:
    """ModelCfg from any object with the synth.ModelConfig fields."""
    return ModelCfg(n_layers=cfg.n_layers, d_model=cfg.d_model, n_heads=cfg.n_heads, n_kv_heads=cfg.n_kv_heads,
                    head_dim=cfg.head_dim, d_ff=cfg.d_ff, vocab=cfg.vocab, mask_id=cfg.vocab - 1,
                    rms_eps=cfg.rms_eps, rope_base=cfg.rope_base,
                    dtype=DLLM_F32 if cfg.dtype == "f32" else DLLM_BF16)


# ---------------------------------------------------------------- objects
class DecodeState:
    """Device tensors of the decoding state (dllm_state)."""

    def __init__(self, B, P, G, device="cuda"):
        L = P + G
        self.B, self.P, self.G = B, P, G
        self.x = torch.zeros((B, L), dtype=torch.int32, device=device)
        self.commit_step = torch.zeros((B, G), dtype=torch.int32, device=device)
        self.reason = torch.zeros((B, G), dtype=torch.int8, device=device)
        self.s = torch.zeros((B, G), dtype=torch.float32, device=device)
        self.budget = torch.zeros((B, G), dtype=torch.int32, device=device)
        self.ell = torch.zeros((B,), dtype=torch.int32, device=device)
        self.done = torch.zeros((B,), dtype=torch.int32, device=device)

    def c(self) -> State:
        return State(*[t.data_ptr() for t in (self.x, self.commit_step, self.reason, self.s, self.budget, self.ell,
                                               self.done)])

    def snapshot(self):
        return {k: getattr(self, k).clone() for k in ("x", "commit_step", "reason", "s", "budget", "ell", "done")}

    def restore(self, snap):
        for k, v in snap.items():
            getattr(self, k).copy_(v)


class Model:
    """A model handle over caller-owned device weights and model buffer (both
    kept alive here).  The LM-head copy is written on the current stream."""

    def __init__(self, cfg, weights, stream=None):
        L = lib()
        self.cfg = cfg
        self.mask_id = cfg.vocab - 1
        self.weights = list(weights)
        self._c = model_cfg(cfg)
        n = ctypes.c_size_t()
        check(L.dllm_model_buffer_size(ctypes.byref(self._c), ctypes.byref(n)))
        dev = self.weights[0].device
        self.model_buf = device_buffer(n.value, dev) if n.value else None
        self.packed_buf = None
        arr = (ctypes.c_void_p * len(self.weights))(*[w.data_ptr() for w in self.weights])
        h = ctypes.c_void_p()
        check(L.dllm_model_create(ctypes.byref(self._c), arr, len(self.weights), _ptr(self.model_buf), n.value,
                                  _stream(stream), ctypes.byref(h)))
        self.h = h

    def packed_size(self):
        n = ctypes.c_size_t()
        check(lib().dllm_model_packed_size(self.h, ctypes.byref(n)))
        return n.value

    def pack_weights(self, stream=None):
        """dllm_model_pack_weights: tiled copies of the projection weights for the
        block-row GEMMs, in a buffer allocated here (once)."""
        if self.packed_buf is None:
            n = self.packed_size()
            buf = device_buffer(n, self.weights[0].device)
            check(lib().dllm_model_pack_weights(self.h, _ptr(buf), n, _stream(stream)))
            self.packed_buf = buf
        return self

    def close(self):
        if getattr(self, "h", None):
            lib().dllm_model_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # workspace --------------------------------------------------------------
    def workspace_size(self, B, L, rows):
        n = ctypes.c_size_t()
        check(lib().dllm_workspace_size(self.h, B, L, rows, ctypes.byref(n)))
        return n.value

    def workspace(self, B, L, rows, device="cuda"):
        return device_buffer(self.workspace_size(B, L, rows), device)

    def layout(self, B, L, rows) -> WsLayout:
        out = WsLayout()
        check(lib().dllm_workspace_layout(self.h, B, L, rows, ctypes.byref(out)))
        return out

    # stages -----------------------------------------------------------------
    def embed(self, x, ws, stream=None):
        B, L = x.shape
        check(lib().dllm_embed(self.h, _ptr(x), B, L, _ptr(ws), ws.numel(), _stream(stream)))

    def layer(self, layer, part, B, L, ws, stream=None):
        check(lib().dllm_layer(self.h, layer, part, B, L, _ptr(ws), ws.numel(), _stream(stream)))

    def head(self, B, L, row0, rows, ws, logits=False, stream=None):
        dev = ws.device
        conf = torch.empty((B * rows,), dtype=torch.float32, device=dev)
        arg = torch.empty((B * rows,), dtype=torch.int32, device=dev)
        lg = torch.empty((B * rows, self.cfg.vocab), dtype=torch.float32, device=dev) if logits else None
        check(lib().dllm_head(self.h, B, L, row0, rows, _ptr(conf), _ptr(arg), _ptr(lg), _ptr(ws), ws.numel(),
                              _stream(stream)))
        return conf.view(B, rows), arg.view(B, rows), (lg.view(B, rows, -1) if logits else None)

    def head_noalloc(self, h, B, L, row0, rows, logits=False, stream=None):
        """dllm_head_noalloc on the caller's residual h (float32 [B*L, d])."""
        dev = h.device
        conf = torch.empty((B * rows,), dtype=torch.float32, device=dev)
        arg = torch.empty((B * rows,), dtype=torch.int32, device=dev)
        lg = torch.empty((B * rows, self.cfg.vocab), dtype=torch.float32, device=dev) if logits else None
        check(lib().dllm_head_noalloc(self.h, _ptr(h), B, L, row0, rows, _ptr(conf), _ptr(arg), _ptr(lg),
                                      _stream(stream)))
        return conf.view(B, rows), arg.view(B, rows), (lg.view(B, rows, -1) if logits else None)

    def forward(self, x, row0, rows, ws=None, logits=False, stream=None):
        B, L = x.shape
        ws = ws if ws is not None else self.workspace(B, L, rows, x.device)
        dev = x.device
        conf = torch.empty((B * rows,), dtype=torch.float32, device=dev)
        arg = torch.empty((B * rows,), dtype=torch.int32, device=dev)
        lg = torch.empty((B * rows, self.cfg.vocab), dtype=torch.float32, device=dev) if logits else None
        check(lib().dllm_forward(self.h, _ptr(x), B, L, row0, rows, _ptr(conf), _ptr(arg), _ptr(lg), _ptr(ws),
                                 ws.numel(), _stream(stream)))
        return conf.view(B, rows), arg.view(B, rows), (lg.view(B, rows, -1) if logits else None)

    # decoding ---------------------------------------------------------------
    def state_init(self, prompt, G, st: DecodeState, stream=None):
        state_init(self.mask_id, prompt, G, st, stream)

    def step(self, ctl: Controller, st: DecodeState, block, t, ws, record=False, wait=True, stream=None):
        p = ctl.to_c()
        c = st.c()
        B, bl = st.B, ctl.block_len
        conf = torch.empty((B, bl), dtype=torch.float32, device=st.x.device) if record else None
        arg = torch.empty((B, bl), dtype=torch.int32, device=st.x.device) if record else None
        flag = torch.zeros((1,), dtype=torch.int32).pin_memory() if wait else None
        check(lib().dllm_step(self.h, ctypes.byref(p), ctypes.byref(c), B, st.P, st.G, block, t, _ptr(conf),
                              _ptr(arg), _ptr(flag), _ptr(ws), ws.numel(), _stream(stream)))
        return (int(flag.item()) if wait else None), conf, arg

    def generate(self, ctl: Controller, prompt, G, ws=None, st=None, trace=False, stream=None):
        B, P = prompt.shape
        bl, T = ctl.block_len, ctl.T
        nb = G // bl
        st = st or DecodeState(B, P, G, prompt.device)
        ws = ws if ws is not None else self.workspace(B, P + G, bl, prompt.device)
        p = ctl.to_c()
        c = st.c()
        fwd = (ctypes.c_int32 * nb)()
        tot = ctypes.c_int32()
        ct = at = None
        if trace:
            ct = torch.full((nb, T, B, bl), float("nan"), dtype=torch.float32, device=prompt.device)
            at = torch.full((nb, T, B, bl), -1, dtype=torch.int32, device=prompt.device)
        check(lib().dllm_generate(self.h, ctypes.byref(p), _ptr(prompt), B, P, G, ctypes.byref(c), fwd,
                                  ctypes.byref(tot), _ptr(ct), _ptr(at), _ptr(ws), ws.numel(), _stream(stream)))
        return GenResult(st, list(fwd), tot.value, ct, at)

    # cross-step key/value reuse ---------------------------------------------
    def kv_cache(self, B, L, device="cuda"):
        """A caller-owned, 256-byte aligned cache buffer for B sequences of L positions."""
        n = ctypes.c_size_t()
        check(lib().dllm_kv_cache_size(self.h, B, L, ctypes.byref(n)))
        return device_buffer(n.value, device)

    def forward_kv(self, x, row0, rows, kv, refresh, ws=None, logits=False, stream=None):
        """dllm_forward_kv: the refresh forward (refresh=True) or the cached forward of rows [row0, row0 + rows)."""
        B, L = x.shape
        ws = ws if ws is not None else self.workspace(B, L, rows, x.device)
        dev = x.device
        conf = torch.empty((B * rows,), dtype=torch.float32, device=dev)
        arg = torch.empty((B * rows,), dtype=torch.int32, device=dev)
        lg = torch.empty((B * rows, self.cfg.vocab), dtype=torch.float32, device=dev) if logits else None
        check(lib().dllm_forward_kv(self.h, _ptr(x), B, L, row0, rows, int(bool(refresh)), _ptr(conf), _ptr(arg),
                                    _ptr(lg), _ptr(kv), kv.numel(), _ptr(ws), ws.numel(), _stream(stream)))
        return conf.view(B, rows), arg.view(B, rows), (lg.view(B, rows, -1) if logits else None)

    def embed_rows(self, x, row0, rows, ws, stream=None):
        B, L = x.shape
        check(lib().dllm_embed_rows(self.h, _ptr(x), B, L, row0, rows, _ptr(ws), ws.numel(), _stream(stream)))

    def layer_kv(self, layer, part, B, L, row0, rows, kv, ws, stream=None):
        check(lib().dllm_layer_kv(self.h, layer, part, B, L, row0, rows, _ptr(kv), kv.numel(), _ptr(ws), ws.numel(),
                                  _stream(stream)))

    def step_kv(self, ctl: Controller, st: DecodeState, block, t, refresh, kv, ws, record=False, wait=True,
                stream=None):
        p = ctl.to_c()
        c = st.c()
        B, bl = st.B, ctl.block_len
        conf = torch.empty((B, bl), dtype=torch.float32, device=st.x.device) if record else None
        arg = torch.empty((B, bl), dtype=torch.int32, device=st.x.device) if record else None
        flag = torch.zeros((1,), dtype=torch.int32).pin_memory() if wait else None
        check(lib().dllm_step_kv(self.h, ctypes.byref(p), int(bool(refresh)), ctypes.byref(c), B, st.P, st.G, block,
                                 t, _ptr(conf), _ptr(arg), _ptr(flag), _ptr(kv), kv.numel(), _ptr(ws), ws.numel(),
                                 _stream(stream)))
        return (int(flag.item()) if wait else None), conf, arg

    def generate_kv(self, ctl: Controller, prompt, G, refresh_every, ws=None, st=None, kv=None, trace=False,
                    stream=None):
        """dllm_generate_kv: the decode with the cache refreshed at steps t % refresh_every == 0."""
        B, P = prompt.shape
        bl, T = ctl.block_len, ctl.T
        nb = G // bl
        st = st or DecodeState(B, P, G, prompt.device)
        ws = ws if ws is not None else self.workspace(B, P + G, bl, prompt.device)
        kv = kv if kv is not None else self.kv_cache(B, P + G, prompt.device)
        p = ctl.to_c()
        c = st.c()
        fwd = (ctypes.c_int32 * nb)()
        tot = ctypes.c_int32()
        ct = at = None
        if trace:
            ct = torch.full((nb, T, B, bl), float("nan"), dtype=torch.float32, device=prompt.device)
            at = torch.full((nb, T, B, bl), -1, dtype=torch.int32, device=prompt.device)
        check(lib().dllm_generate_kv(self.h, ctypes.byref(p), refresh_every, _ptr(prompt), B, P, G, ctypes.byref(c),
                                     fwd, ctypes.byref(tot), _ptr(ct), _ptr(at), _ptr(kv), kv.numel(), _ptr(ws),
                                     ws.numel(), _stream(stream)))
        return GenResult(st, list(fwd), tot.value, ct, at)

    # profiling --------------------------------------------------------------
    def prof_enable(self, kinds=()):
        """Record per-launch HIP-event timings for the given kernel kinds (PROF_*)."""
        mask = 0
        for k in kinds:
            mask |= 1 << k
        check(lib().dllm_prof_enable(self.h, mask))

    def prof_every(self, every):
        """dllm_prof_every: record one launch in `every` of each enabled kind."""
        check(lib().dllm_prof_every(self.h, every))

    def prof_read(self, kind):
        ms = ctypes.c_double()
        n = ctypes.c_int64()
        check(lib().dllm_prof_read(self.h, kind, ctypes.byref(ms), ctypes.byref(n)))
        return ms.value, n.value


@dataclass
class GenResult:
    state: DecodeState
    forwards: list
    total_forwards: int
    conf_trace: torch.Tensor | None
    argmax_trace: torch.Tensor | None


def state_init(mask_id, prompt, G, st: DecodeState, stream=None):
    """dllm_state_init: x = [prompt | mask], commit_step = -1, everything else 0."""
    B, P = prompt.shape
    c = st.c()
    check(lib().dllm_state_init(mask_id, _ptr(prompt), B, P, G, ctypes.byref(c), _stream(stream)))


def commit(ctl: Controller, st: DecodeState, conf, argmax, block, t, mask_id, all_done=None, stream=None):
    """The controller alone (dllm_commit) on device conf [B, bl] / argmax [B, bl]."""
    p = ctl.to_c()
    c = st.c()
    check(lib().dllm_commit(ctypes.byref(p), ctypes.byref(c), _ptr(conf), _ptr(argmax), st.B, st.P, st.G, block, t,
                            mask_id, _ptr(all_done), _stream(stream)))
