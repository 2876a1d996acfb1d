"""Thin ctypes binding of liblodestar.so (include/lodestar.h).

Argument marshalling only: torch tensors are checked for dtype, device, shape
and contiguity, then their data pointers and the current HIP stream are passed
to the C functions of the same name.  Every step of the hot path runs in the
library's HIP kernels.  There is no fallback: if the library is missing the
import of a Context fails loudly.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "liblodestar.so")

LS_OK, LS_ERR_INVALID, LS_ERR_NOMEM, LS_ERR_DEVICE, LS_ERR_STATE, LS_ERR_UNSUPPORTED = 0, -1, -2, -3, -4, -5
LS_FP32, LS_BF16 = 0, 1
DERIVED_COLS = 5
_DTYPES = {"fp32": LS_FP32, "f32": LS_FP32, "bf16": LS_BF16}


class LodestarError(RuntimeError):
    def __init__(self, func, code, msg):
        super().__init__(f"{func} returned {code}: {msg}")
        self.code = code


class ls_model_config(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int32), ("n_hidden", ctypes.c_int32), ("hidden", ctypes.c_int32 * 3),
                ("block_tokens", ctypes.c_int32), ("dtype", ctypes.c_int32)]


LS_HEUR_PREFIX_LOAD, LS_HEUR_PREFIX_THRESHOLD = 1, 2
LS_ROUTE_OK, LS_ROUTE_COLD_START, LS_ROUTE_OOD = 0, 1, 2
LS_ROUTE_EXPLORED, LS_ROUTE_KFILTER, LS_ROUTE_TIEBREAK = 0x100, 0x200, 0x400


class ls_policy(ctypes.Structure):
    _fields_ = [("heuristic", ctypes.c_int32), ("count_cols", ctypes.c_int32 * 2), ("theta_imbal", ctypes.c_float),
                ("overload_k", ctypes.c_float), ("prefix_tau", ctypes.c_float), ("n_samples", ctypes.c_int64),
                ("n_min", ctypes.c_int64), ("lo", ctypes.c_void_p), ("hi", ctypes.c_void_p),
                ("epsilon", ctypes.c_float), ("kv_col", ctypes.c_int32), ("tau_sat", ctypes.c_float),
                ("tau_ben", ctypes.c_float), ("k_filter", ctypes.c_int32), ("delta", ctypes.c_float)]


def make_policy(heuristic=LS_HEUR_PREFIX_LOAD, count_cols=(-1, -1), theta_imbal=0.0, overload_k=0.0, prefix_tau=0.0,
                n_samples=0, n_min=0, lo=None, hi=None, epsilon=0.0, kv_col=-1, tau_sat=0.0, tau_ben=0.0,
                k_filter=0, delta=-1.0):
    """An ls_policy; lo/hi are host float32 arrays of d bounds (kept alive on the returned object)."""
    lo_a = None if lo is None else np.ascontiguousarray(lo, dtype=np.float32)
    hi_a = None if hi is None else np.ascontiguousarray(hi, dtype=np.float32)
    p = ls_policy(int(heuristic), (ctypes.c_int32 * 2)(*count_cols), theta_imbal, overload_k, prefix_tau,
                  int(n_samples), int(n_min), None if lo_a is None else lo_a.ctypes.data,
                  None if hi_a is None else hi_a.ctypes.data, epsilon, int(kv_col), tau_sat, tau_ben, int(k_filter),
                  delta)
    p._bounds = (lo_a, hi_a)
    return p


_lib = None


def library():
    """Load liblodestar.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: run `python -m paper_2606_00946_amd.build` first")
        lib = ctypes.CDLL(LIB_PATH)
        P, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
        cfgp = ctypes.POINTER(ls_model_config)
        lib.ls_param_count.argtypes = [cfgp]
        lib.ls_param_count.restype = i64
        lib.ls_create.argtypes = [cfgp, ctypes.c_int, ctypes.POINTER(P)]
        lib.ls_destroy.argtypes = [P]
        lib.ls_destroy.restype = None
        lib.ls_last_error.argtypes = [P]
        lib.ls_last_error.restype = ctypes.c_char_p
        lib.ls_set_model.argtypes = [P, P, i64, P, P, P]
        lib.ls_get_model.argtypes = [P, P, i64, P, P]
        lib.ls_load_cache_state.argtypes = [P, i32, P, P, P]
        lib.ls_score_batch.argtypes = [P, i32, i32, P, P, P, P, P, P, P, P, P, P]
        lib.ls_update.argtypes = [P, i32, P, P, f32, P, P, P]
        lib.ls_profile_enable.argtypes = [P, ctypes.c_int]
        lib.ls_set_exact_scores.argtypes = [P, ctypes.c_int]
        lib.ls_set_prefix_join.argtypes = [P, ctypes.c_int]
        lib.ls_set_prefix_closed.argtypes = [P, ctypes.c_int]
        lib.ls_buffer_init.argtypes = [P, i32, i32]
        lib.ls_buffer_push.argtypes = [P, i32, P, P, P, P]
        lib.ls_buffer_state.argtypes = [P, P, P, P]
        lib.ls_buffer_read.argtypes = [P, P, P, P, P, P]
        lib.ls_train_round.argtypes = [P, i32, i32, f32, P, P, P]
        lib.ls_route_batch.argtypes = [P, ctypes.POINTER(ls_policy), i32, i32, P, P, P, P, P, P, P, P, P, P]
        lib.ls_profile_read.argtypes = [P, i32, P, P, P, P]
        lib.ls_set_cache_capacity.argtypes = [P, i32, P]
        lib.ls_set_dropout.argtypes = [P, f32, ctypes.c_uint64]
        lib.ls_commit_routes.argtypes = [P, i32, i64, P, P, P, P]
        lib.ls_read_cache_state.argtypes = [P, i32, P, P, P, i64, P]
        lib.ls_set_shadow_training.argtypes = [P, ctypes.c_int, P]
        lib.ls_swap_model.argtypes = [P, P, P]
        lib.ls_fast_scores.argtypes = [P, i32, i32, P, P, P, P, P, P, P, P]
        lib.ls_score_batch_noalloc.argtypes = [P, i32, i32, P, P, P, P, P, P, P, P, P, P]
        lib.ls_set_cu_limit.argtypes = [P, ctypes.c_int]
        lib.ls_set_chain_kernels.argtypes = [P, ctypes.c_int]
        for f in (lib.ls_create, lib.ls_set_model, lib.ls_get_model, lib.ls_load_cache_state, lib.ls_score_batch,
                  lib.ls_update, lib.ls_profile_enable, lib.ls_profile_read, lib.ls_set_exact_scores,
                  lib.ls_set_prefix_join, lib.ls_route_batch, lib.ls_set_prefix_closed, lib.ls_buffer_init,
                  lib.ls_buffer_push, lib.ls_buffer_state, lib.ls_buffer_read, lib.ls_train_round,
                  lib.ls_set_cache_capacity, lib.ls_commit_routes, lib.ls_read_cache_state, lib.ls_set_dropout,
                  lib.ls_set_shadow_training, lib.ls_swap_model, lib.ls_fast_scores, lib.ls_set_cu_limit,
                  lib.ls_set_chain_kernels,
                  lib.ls_score_batch_noalloc):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def make_config(d, hidden, dtype="fp32", block_tokens=16) -> ls_model_config:
    h = list(hidden) + [0] * (3 - len(hidden))
    return ls_model_config(int(d), len(hidden), (ctypes.c_int32 * 3)(*h), int(block_tokens),
                           _DTYPES[dtype] if isinstance(dtype, str) else int(dtype))


def ls_param_count(d, hidden) -> int:
    cfg = make_config(d, hidden)
    return int(library().ls_param_count(ctypes.byref(cfg)))


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(int(stream.cuda_stream))


_EMPTY = {}


def _empty_ptr(device):
    """A valid one-element device buffer standing in for an empty tensor (whose
    data pointer may be NULL); the library never reads it."""
    import torch
    if device not in _EMPTY:
        _EMPTY[device] = torch.zeros(1, dtype=torch.int64, device=device)
    return ctypes.c_void_p(_EMPTY[device].data_ptr())


def _dev(t, name, dtypes, numel=None, allow_none=False):
    """Device pointer of a contiguous CUDA tensor with one of `dtypes`."""
    if t is None:
        if allow_none:
            return None
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype not in dtypes:
        raise ValueError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} has {t.numel()} elements, expected {numel}")
    if t.numel() == 0:
        return _empty_ptr(t.device)
    return ctypes.c_void_p(t.data_ptr())


def _host(a, dtype, numel=None):
    a = np.ascontiguousarray(a, dtype=dtype)
    if numel is not None and a.size != numel:
        raise ValueError(f"expected {numel} elements, got {a.size}")
    return a, a.ctypes.data_as(ctypes.c_void_p)


class Context:
    """One ls_ctx: model, cache state and workspace on one device."""

    def __init__(self, d, hidden, dtype="fp32", block_tokens=16, device=None):
        import torch
        self.lib = library()
        self.cfg = make_config(d, hidden, dtype, block_tokens)
        self.d = int(d)
        self.hidden = tuple(hidden)
        self.n_params = int(self.lib.ls_param_count(ctypes.byref(self.cfg)))
        if self.n_params < 0:
            raise ValueError("invalid model shape")
        self.device = torch.cuda.current_device() if device is None else int(device)
        h = ctypes.c_void_p()
        rc = self.lib.ls_create(ctypes.byref(self.cfg), self.device, ctypes.byref(h))
        if rc != LS_OK:
            raise LodestarError("ls_create", rc, "could not create a context")
        self.h = h
        self.n_instances = None

    def close(self):
        if getattr(self, "h", None):
            self.lib.ls_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _check(self, func, rc):
        if rc != LS_OK:
            raise LodestarError(func, rc, self.lib.ls_last_error(self.h).decode())
        return rc

    def last_error(self) -> str:
        return self.lib.ls_last_error(self.h).decode()

    # -- model -------------------------------------------------------------
    def ls_set_model(self, params, mu, inv_sigma, stream=None):
        p, pp = _host(params, np.float32, self.n_params)
        m, mp = _host(mu, np.float32, self.d)
        s, sp = _host(inv_sigma, np.float32, self.d)
        return self._check("ls_set_model", self.lib.ls_set_model(self.h, pp, self.n_params, mp, sp, _stream(stream)))

    def ls_get_model(self):
        p = np.zeros(self.n_params, np.float32)
        m = np.zeros(self.d, np.float32)
        s = np.zeros(self.d, np.float32)
        self._check("ls_get_model", self.lib.ls_get_model(self.h, p.ctypes.data_as(ctypes.c_void_p), self.n_params,
                                                          m.ctypes.data_as(ctypes.c_void_p),
                                                          s.ctypes.data_as(ctypes.c_void_p)))
        return p, m, s

    # -- cache state -------------------------------------------------------
    def ls_load_cache_state(self, inst_off, hashes, stream=None):
        import torch
        off, offp = _host(inst_off, np.int64)
        N = off.size - 1
        hp = _dev(hashes, "hashes", (torch.int64, torch.uint64), int(off[-1]) if N >= 0 else None)
        rc = self.lib.ls_load_cache_state(self.h, N, offp, hp, _stream(stream))
        self._check("ls_load_cache_state", rc)
        self.n_instances = N
        return rc

    def ls_set_shadow_training(self, enable=True, stream=None):
        """Double-buffered retraining: updates act on a shadow copy of the model."""
        return self._check("ls_set_shadow_training",
                           self.lib.ls_set_shadow_training(self.h, int(bool(enable)), _stream(stream)))

    def ls_swap_model(self, serve_stream=None, train_stream=None):
        """Make the shadow model the live one (ordered between the two streams)."""
        return self._check("ls_swap_model",
                           self.lib.ls_swap_model(self.h, _stream(serve_stream), _stream(train_stream)))

    def ls_set_dropout(self, p, seed=0):
        """Dropout rate p in [0, 1) on the hidden activations of later updates (0: off)."""
        return self._check("ls_set_dropout", self.lib.ls_set_dropout(self.h, float(p), ctypes.c_uint64(int(seed))))

    # -- prefix-index maintenance -----------------------------------------
    def ls_set_cache_capacity(self, capacity):
        """capacity: per-instance blocks (host array), or None to turn maintenance off."""
        if capacity is None:
            return self._check("ls_set_cache_capacity", self.lib.ls_set_cache_capacity(self.h, 0, None))
        cap, capp = _host(capacity, np.int64)
        return self._check("ls_set_cache_capacity", self.lib.ls_set_cache_capacity(self.h, cap.size, capp))

    def ls_commit_routes(self, req_off, req_hashes, chosen, n_hashes=None, stream=None):
        """Records a routed batch; n_hashes defaults to req_off[-1] (read from the device)."""
        import torch
        R = req_off.numel() - 1
        if n_hashes is None:
            n_hashes = int(req_off[-1].item()) if R >= 0 else 0
        op = _dev(req_off, "req_off", (torch.int64,), R + 1)
        hp = _dev(req_hashes, "req_hashes", (torch.int64, torch.uint64), n_hashes)
        cp = _dev(chosen, "chosen", (torch.int32,), R)
        return self._check("ls_commit_routes",
                           self.lib.ls_commit_routes(self.h, R, int(n_hashes), op, hp, cp, _stream(stream)))

    def ls_read_cache_state(self, stream=None):
        """(inst_off numpy int64 [N+1], hashes int64 tensor, stamps int64 tensor) of the maintained lists."""
        import torch
        N = self.n_instances
        off = np.zeros(N + 1, np.int64)
        offp = off.ctypes.data_as(ctypes.c_void_p)
        self._check("ls_read_cache_state", self.lib.ls_read_cache_state(self.h, N, offp, None, None, 0,
                                                                         _stream(stream)))
        total = int(off[-1])
        h = torch.empty(max(total, 1), dtype=torch.int64, device="cuda")
        st = torch.empty(max(total, 1), dtype=torch.int64, device="cuda")
        self._check("ls_read_cache_state",
                    self.lib.ls_read_cache_state(self.h, N, offp, ctypes.c_void_p(h.data_ptr()),
                                                 ctypes.c_void_p(st.data_ptr()), h.numel(), _stream(stream)))
        return off, h[:total], st[:total]

    # -- scoring -----------------------------------------------------------
    def ls_score_batch(self, req_off, req_hashes, prompt_len, inst_feat, chosen, min_ttft=None, scores=None,
                       overlap=None, feat_out=None, stream=None):
        import torch
        R = req_off.numel() - 1
        N = inst_feat.shape[0] if inst_feat.dim() == 2 else (self.n_instances or 0)
        d_inst = self.d - DERIVED_COLS
        args = [
            _dev(req_off, "req_off", (torch.int64,), R + 1),
            _dev(req_hashes, "req_hashes", (torch.int64, torch.uint64)),
            _dev(prompt_len, "prompt_len", (torch.int32,), R),
            _dev(inst_feat, "inst_feat", (torch.float32,), N * d_inst),
            _dev(chosen, "chosen", (torch.int32,), R),
            _dev(min_ttft, "min_ttft", (torch.float32,), R, allow_none=True),
            _dev(scores, "scores", (torch.float32,), R * N, allow_none=True),
            _dev(overlap, "overlap", (torch.int32,), R * N, allow_none=True),
            _dev(feat_out, "feat_out", (torch.float32,), R * self.d, allow_none=True),
        ]
        return self._check("ls_score_batch", self.lib.ls_score_batch(self.h, R, N, *args, _stream(stream)))

    def ls_score_batch_noalloc(self, req_off, req_hashes, prompt_len, inst_feat, chosen, min_ttft=None, scores=None,
                               overlap=None, feat_out=None, stream=None):
        import torch
        R = req_off.numel() - 1
        N = inst_feat.shape[0] if inst_feat.dim() == 2 else (self.n_instances or 0)
        d_inst = self.d - DERIVED_COLS
        args = [
            _dev(req_off, "req_off", (torch.int64,), R + 1),
            _dev(req_hashes, "req_hashes", (torch.int64, torch.uint64)),
            _dev(prompt_len, "prompt_len", (torch.int32,), R),
            _dev(inst_feat, "inst_feat", (torch.float32,), N * d_inst),
            _dev(chosen, "chosen", (torch.int32,), R),
            _dev(min_ttft, "min_ttft", (torch.float32,), R, allow_none=True),
            _dev(scores, "scores", (torch.float32,), R * N, allow_none=True),
            _dev(overlap, "overlap", (torch.int32,), R * N, allow_none=True),
            _dev(feat_out, "feat_out", (torch.float32,), R * self.d, allow_none=True),
        ]
        return self._check("ls_score_batch_noalloc",
                           self.lib.ls_score_batch_noalloc(self.h, R, N, *args, _stream(stream)))

    def ls_route_batch(self, policy, req_off, req_hashes, prompt_len, inst_feat, rnd, chosen, status=None, heur=None,
                       feat_out=None, stream=None):
        import torch
        R = req_off.numel() - 1
        N = inst_feat.shape[0] if inst_feat.dim() == 2 else (self.n_instances or 0)
        d_inst = self.d - DERIVED_COLS
        args = [
            _dev(req_off, "req_off", (torch.int64,), R + 1),
            _dev(req_hashes, "req_hashes", (torch.int64, torch.uint64)),
            _dev(prompt_len, "prompt_len", (torch.int32,), R),
            _dev(inst_feat, "inst_feat", (torch.float32,), N * d_inst),
            _dev(rnd, "rnd", (torch.int32, torch.uint32), 3 * R, allow_none=True),
            _dev(chosen, "chosen", (torch.int32,), R),
            _dev(status, "status", (torch.int32,), R, allow_none=True),
            _dev(heur, "heur", (torch.int32,), R, allow_none=True),
            _dev(feat_out, "feat_out", (torch.float32,), R * self.d, allow_none=True),
        ]
        return self._check("ls_route_batch",
                           self.lib.ls_route_batch(self.h, ctypes.byref(policy), R, N, *args, _stream(stream)))

    # -- online-learning data path -----------------------------------------
    def ls_buffer_init(self, fifo_cap, replay_cap):
        return self._check("ls_buffer_init", self.lib.ls_buffer_init(self.h, int(fifo_cap), int(replay_cap)))

    def ls_buffer_push(self, feats, ttft, admitted=None, stream=None):
        import torch
        B = ttft.numel()
        args = [_dev(feats, "feats", (torch.float32,), B * self.d), _dev(ttft, "ttft", (torch.float32,), B),
                _dev(admitted, "admitted", (torch.int32,), 1, allow_none=True)]
        return self._check("ls_buffer_push", self.lib.ls_buffer_push(self.h, B, *args, _stream(stream)))

    def ls_buffer_state(self):
        v = [ctypes.c_int32(0) for _ in range(3)]
        self._check("ls_buffer_state", self.lib.ls_buffer_state(self.h, *[ctypes.byref(x) for x in v]))
        return tuple(x.value for x in v)          # (fifo_count, fifo_head, replay_count)

    def ls_buffer_read(self, stream=None):
        """Device copies of the FIFO (oldest first) and the pool (by slot)."""
        import torch
        fc, _, rc = self.ls_buffer_state()
        fx = torch.empty(max(fc, 1) * self.d, dtype=torch.float32, device="cuda")
        fy = torch.empty(max(fc, 1), dtype=torch.float32, device="cuda")
        rx = torch.empty(max(rc, 1) * self.d, dtype=torch.float32, device="cuda")
        ry = torch.empty(max(rc, 1), dtype=torch.float32, device="cuda")
        self._check("ls_buffer_read", self.lib.ls_buffer_read(self.h, ctypes.c_void_p(fx.data_ptr()),
                                                              ctypes.c_void_p(fy.data_ptr()),
                                                              ctypes.c_void_p(rx.data_ptr()),
                                                              ctypes.c_void_p(ry.data_ptr()), _stream(stream)))
        return (fx[:fc * self.d].view(fc, self.d), fy[:fc], rx[:rc * self.d].view(rc, self.d), ry[:rc])

    def ls_train_round(self, epochs, batch, lr, perm=None, loss_out=None, stream=None):
        import torch
        pa = None if perm is None else np.ascontiguousarray(perm, dtype=np.int32)
        lo = _dev(loss_out, "loss_out", (torch.float32,), 1, allow_none=True)
        return self._check("ls_train_round",
                           self.lib.ls_train_round(self.h, int(epochs), int(batch), float(lr),
                                                   None if pa is None else pa.ctypes.data_as(ctypes.c_void_p), lo,
                                                   _stream(stream)))

    # -- online update -----------------------------------------------------
    def ls_update(self, feats, ttft, lr, loss_out=None, grad_out=None, stream=None):
        import torch
        B = ttft.numel()
        args = [
            _dev(feats, "feats", (torch.float32,), B * self.d),
            _dev(ttft, "ttft", (torch.float32,), B),
        ]
        lo = _dev(loss_out, "loss_out", (torch.float32,), 1, allow_none=True)
        go = _dev(grad_out, "grad_out", (torch.float32,), self.n_params, allow_none=True)
        return self._check("ls_update", self.lib.ls_update(self.h, B, *args, float(lr), lo, go, _stream(stream)))

    def ls_set_chain_kernels(self, mode):
        return self._check("ls_set_chain_kernels", self.lib.ls_set_chain_kernels(self.h, int(mode)))

    def ls_set_exact_scores(self, enable=True):
        return self._check("ls_set_exact_scores", self.lib.ls_set_exact_scores(self.h, 1 if enable else 0))

    def ls_fast_scores(self, req_off, req_hashes, prompt_len, inst_feat, t, err, band=None, stream=None):
        import torch
        R = req_off.numel() - 1
        N = inst_feat.shape[0] if inst_feat.dim() == 2 else (self.n_instances or 0)
        d_inst = self.d - DERIVED_COLS
        args = [
            _dev(req_off, "req_off", (torch.int64,), R + 1),
            _dev(req_hashes, "req_hashes", (torch.int64, torch.uint64)),
            _dev(prompt_len, "prompt_len", (torch.int32,), R),
            _dev(inst_feat, "inst_feat", (torch.float32,), N * d_inst),
            _dev(t, "t", (torch.float32,), R * N),
            _dev(err, "err", (torch.float32,), R * N),
            _dev(band, "band", (torch.uint8,), R * N, allow_none=True),
        ]
        return self._check("ls_fast_scores", self.lib.ls_fast_scores(self.h, R, N, *args, _stream(stream)))

    def ls_set_cu_limit(self, n=0):
        return self._check("ls_set_cu_limit", self.lib.ls_set_cu_limit(self.h, int(n)))

    def ls_set_prefix_closed(self, enable=True):
        return self._check("ls_set_prefix_closed", self.lib.ls_set_prefix_closed(self.h, 1 if enable else 0))

    def ls_set_prefix_join(self, mode=0):
        return self._check("ls_set_prefix_join", self.lib.ls_set_prefix_join(self.h, int(mode)))

    # -- per-kernel timing ------------------------------------------------
    def ls_profile_enable(self, enable=True):
        return self._check("ls_profile_enable", self.lib.ls_profile_enable(self.h, 1 if enable else 0))

    def ls_profile_read(self) -> dict:
        """{kind: (launches, total_ms)} since profiling was enabled (synchronous)."""
        k = 16
        names = (ctypes.c_char_p * k)()
        launches = (ctypes.c_int64 * k)()
        ms = (ctypes.c_double * k)()
        n = ctypes.c_int32()
        self._check("ls_profile_read", self.lib.ls_profile_read(self.h, k, names, launches, ms, ctypes.byref(n)))
        return {names[i].decode(): (int(launches[i]), float(ms[i])) for i in range(min(k, n.value))}
