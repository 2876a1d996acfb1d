"""CPU oracle for the batched routing scorer -- test infrastructure only.

A ctypes front end for ``lodestar_oracle.c``.  Only the tests, the smoke check
and the benchmark's CPU-baseline leg use it; the HIP library never does, and
the two share no code.  Every function is a plain transcription of what the
paper defines (see the C file for the passages each one follows).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

F64, F32, BF16 = 0, 1, 2
MODES = {"f64": F64, "fp32": F32, "f32": F32, "bf16": BF16}

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lodestar_oracle.c")
_LIB = os.path.join(_HERE, "liblsoracle.so")
_CFLAGS = ["-O2", "-mfma", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-shared", "-fPIC", "-std=c11"]


# The same source with AddressSanitizer and UndefinedBehaviorSanitizer (any
# finding aborts); a process loads it with both runtimes preloaded.
SANITIZE_FLAGS = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                  "-fno-omit-frame-pointer"]


def compile_c(src: str, out: str, extra=()) -> str:
    tmp = f"{out}.{os.getpid()}.tmp"
    flags = [f for f in _CFLAGS if not (extra and f.startswith("-O"))]
    subprocess.check_call(["gcc", *flags, *extra, "-o", tmp, src, "-lm"])
    os.replace(tmp, out)
    return out


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (no GPU code involved)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        compile_c(_SRC, _LIB)
    return _LIB


_libs = {}


def _open(path):
    if path not in _libs:
        lib = ctypes.CDLL(path)
        P = ctypes.c_void_p
        i32, i64, f32, dbl = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double
        lib.lso_bf16_round.argtypes = [f32]
        lib.lso_bf16_round.restype = f32
        lib.lso_overlap.argtypes = [i32, P, P, P, i32, P, P, P, ctypes.c_int]
        lib.lso_features.argtypes = [ctypes.c_int, i32, P, i32, i32, i32, P]
        lib.lso_param_count.argtypes = [i32, i32, P]
        lib.lso_param_count.restype = i64
        lib.lso_forward.argtypes = [ctypes.c_int, i32, i32, P, P, P, P, i64, P, P, ctypes.c_int]
        lib.lso_argmin.argtypes = [i32, P, P]
        lib.lso_argmin.restype = i32
        lib.lso_score.argtypes = [ctypes.c_int, i32, i32, P, P, P, P, i32, P, P, P, P, i32, P, P, P,
                                  P, P, P, P, P, ctypes.c_int]
        lib.lso_update.argtypes = [ctypes.c_int, i32, i32, P, P, P, P, i32, P, P, f32, P, P]
        lib.lso_splitmix64_mix.argtypes = [ctypes.c_uint64]
        lib.lso_splitmix64_mix.restype = ctypes.c_uint64
        lib.lso_hrw_topk.argtypes = [i32, ctypes.c_uint64, i32, P]
        lib.lso_hrw_topk.restype = i32
        lib.lso_heuristic.argtypes = [i32, i32, P, P, dbl, dbl, dbl]
        lib.lso_heuristic.restype = i32
        lib.lso_route.argtypes = [ctypes.c_int, i32, i32, P, P, P, P, i32, P, P, P, P, i32, P, P, P,
                                  ctypes.POINTER(Policy), P, P, P, P, ctypes.c_int]
        lib.lso_embed.argtypes = [ctypes.c_int, i32, i32, P, P, P, P, i32, P, P, P]
        lib.lso_buffer_push.argtypes = [ctypes.c_int, i32, i32, P, P, P, P, i32, i32, P, P, P, P, P, P, P, i32, P, P,
                                        P]
        lib.lso_train_round.argtypes = [ctypes.c_int, i32, i32, P, P, P, P, i32, i32, i32, P, P, i32, P, P, i32, i32,
                                        f32, P, P]
        u64 = ctypes.c_uint64
        lib.lso_update_dropout.argtypes = [ctypes.c_int, i32, i32, P, P, P, P, i32, P, P, f32, dbl, u64, u64, P, P]
        lib.lso_train_round_dropout.argtypes = [ctypes.c_int, i32, i32, P, P, P, P, i32, i32, i32, P, P, i32, P, P,
                                                i32, i32, f32, P, dbl, u64, u64, P]
        lib.lso_stamp.argtypes = [ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32]
        lib.lso_stamp.restype = ctypes.c_uint64
        lib.lso_commit.argtypes = [i32, P, P, P, P, i32, P, P, P, ctypes.c_uint32, P, P, P]
        for f in (lib.lso_overlap, lib.lso_forward, lib.lso_score, lib.lso_update, lib.lso_route, lib.lso_embed,
                  lib.lso_buffer_push, lib.lso_train_round, lib.lso_commit, lib.lso_update_dropout,
                  lib.lso_train_round_dropout):
            f.restype = ctypes.c_int
        _libs[path] = lib
    return _libs[path]


class Policy(ctypes.Structure):
    """Routing-policy parameters (mirrors lso_policy in the C file)."""
    _fields_ = [("heuristic", ctypes.c_int32), ("count_col0", ctypes.c_int32), ("count_col1", ctypes.c_int32),
                ("kv_col", ctypes.c_int32), ("k_filter", ctypes.c_int32), ("pad", ctypes.c_int32),
                ("theta_imbal", ctypes.c_double), ("overload_k", ctypes.c_double), ("prefix_tau", ctypes.c_double),
                ("n_samples", ctypes.c_int64), ("n_min", ctypes.c_int64),
                ("epsilon", ctypes.c_double), ("tau_sat", ctypes.c_double), ("tau_ben", ctypes.c_double),
                ("delta", ctypes.c_double), ("lo", ctypes.c_void_p), ("hi", ctypes.c_void_p)]


ROUTE_OK, ROUTE_COLD_START, ROUTE_OOD = 0, 1, 2
ROUTE_EXPLORED, ROUTE_KFILTER, ROUTE_TIEBREAK = 0x100, 0x200, 0x400

_active = None


def _load():
    if _active is not None:
        return _open(_active)
    return _open(build())


def use_library(path) -> None:
    """Point this module at another build of the oracle source (None: the default)."""
    global _active
    _active = path


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _mode(m):
    return MODES[m] if isinstance(m, str) else int(m)


def bf16_round(x) -> np.ndarray:
    lib = _load()
    x = np.asarray(x, dtype=np.float32)
    return np.array([lib.lso_bf16_round(float(v)) for v in x.ravel()], dtype=np.float32).reshape(x.shape)


def overlap(req_off, req_hashes, inst_off, inst_hashes, sel=None, threads=0) -> np.ndarray:
    lib = _load()
    req_off = _c(req_off, np.int64); req_hashes = _c(req_hashes, np.uint64)
    inst_off = _c(inst_off, np.int64); inst_hashes = _c(inst_hashes, np.uint64)
    N = inst_off.shape[0] - 1
    R = req_off.shape[0] - 1
    sel_a = None if sel is None else _c(sel, np.int32)
    n_sel = R if sel_a is None else sel_a.shape[0]
    out = np.zeros((n_sel, N), dtype=np.int32)
    rc = lib.lso_overlap(n_sel, _ptr(sel_a), _ptr(req_off), _ptr(req_hashes), N, _ptr(inst_off),
                         _ptr(inst_hashes), _ptr(out), threads)
    assert rc == 0, rc
    return out


def features(mode, inst_row, L, n, l) -> np.ndarray:
    lib = _load()
    inst_row = _c(inst_row, np.float32)
    x = np.zeros(inst_row.shape[0] + 5, dtype=np.float64)
    lib.lso_features(_mode(mode), inst_row.shape[0], _ptr(inst_row), int(L), int(n), int(l), _ptr(x))
    return x


def param_count(d, hidden) -> int:
    lib = _load()
    h = _c(hidden, np.int32)
    return int(lib.lso_param_count(d, h.shape[0], _ptr(h)))


def forward(mode, d, hidden, params, mu, inv_sigma, x, threads=0) -> np.ndarray:
    lib = _load()
    h = _c(hidden, np.int32)
    params = _c(params, np.float32); mu = _c(mu, np.float32); inv_sigma = _c(inv_sigma, np.float32)
    x = _c(x, np.float64).reshape(-1, d)
    out = np.zeros(x.shape[0], dtype=np.float64)
    rc = lib.lso_forward(_mode(mode), d, h.shape[0], _ptr(h), _ptr(params), _ptr(mu), _ptr(inv_sigma),
                         x.shape[0], _ptr(x), _ptr(out), threads)
    assert rc == 0, rc
    return out


def argmin(scores):
    lib = _load()
    s = _c(scores, np.float64)
    m = np.zeros(1, dtype=np.float64)
    i = lib.lso_argmin(s.shape[0], _ptr(s), _ptr(m))
    return int(i), float(m[0])


def score(mode, d, hidden, params, mu, inv_sigma, req_off, req_hashes, prompt_len, inst_feat,
          inst_off, inst_hashes, sel=None, threads=0) -> dict:
    """Overlap, features, model and argmin for the selected requests."""
    lib = _load()
    h = _c(hidden, np.int32)
    params = _c(params, np.float32); mu = _c(mu, np.float32); inv_sigma = _c(inv_sigma, np.float32)
    req_off = _c(req_off, np.int64); req_hashes = _c(req_hashes, np.uint64)
    prompt_len = _c(prompt_len, np.int32); inst_feat = _c(inst_feat, np.float32)
    inst_off = _c(inst_off, np.int64); inst_hashes = _c(inst_hashes, np.uint64)
    N = inst_off.shape[0] - 1
    R = req_off.shape[0] - 1
    sel_a = None if sel is None else _c(sel, np.int32)
    n_sel = R if sel_a is None else sel_a.shape[0]
    ov = np.zeros((n_sel, N), dtype=np.int32)
    sc = np.zeros((n_sel, N), dtype=np.float64)
    ch = np.zeros(n_sel, dtype=np.int32)
    mn = np.zeros(n_sel, dtype=np.float64)
    ft = np.zeros((n_sel, d), dtype=np.float64)
    rc = lib.lso_score(_mode(mode), d, h.shape[0], _ptr(h), _ptr(params), _ptr(mu), _ptr(inv_sigma),
                       n_sel, _ptr(sel_a), _ptr(req_off), _ptr(req_hashes), _ptr(prompt_len), N,
                       _ptr(inst_feat), _ptr(inst_off), _ptr(inst_hashes),
                       _ptr(ov), _ptr(sc), _ptr(ch), _ptr(mn), _ptr(ft), threads)
    assert rc == 0, rc
    return {"overlap": ov, "scores": sc, "chosen": ch, "min_ttft": mn, "feat": ft}


def update(mode, d, hidden, params, mu, inv_sigma, feats, ttft, lr, dropout=None) -> dict:
    """One SGD step; returns the new params, the gradient and the pre-step loss.
    dropout: None, or (p, seed, step) -- the masks of update call `step`."""
    lib = _load()
    h = _c(hidden, np.int32)
    p = np.array(params, dtype=np.float32, copy=True)
    mu = _c(mu, np.float32); inv_sigma = _c(inv_sigma, np.float32)
    feats = _c(feats, np.float32).reshape(-1, d); ttft = _c(ttft, np.float32)
    grad = np.zeros(p.shape[0], dtype=np.float64)
    loss = np.zeros(1, dtype=np.float64)
    if dropout is None:
        rc = lib.lso_update(_mode(mode), d, h.shape[0], _ptr(h), _ptr(p), _ptr(mu), _ptr(inv_sigma),
                            feats.shape[0], _ptr(feats), _ptr(ttft), float(lr), _ptr(grad), _ptr(loss))
    else:
        dp, seed, step = dropout
        rc = lib.lso_update_dropout(_mode(mode), d, h.shape[0], _ptr(h), _ptr(p), _ptr(mu), _ptr(inv_sigma),
                                    feats.shape[0], _ptr(feats), _ptr(ttft), float(lr), float(dp),
                                    ctypes.c_uint64(seed), ctypes.c_uint64(step), _ptr(grad), _ptr(loss))
    assert rc == 0, rc
    return {"params": p, "grad": grad, "loss": float(loss[0])}


def splitmix64_mix(z: int) -> int:
    return int(_load().lso_splitmix64_mix(ctypes.c_uint64(z & 0xFFFFFFFFFFFFFFFF)))


def hrw_topk(N: int, key: int, K: int) -> np.ndarray:
    out = np.zeros(max(K, 1), dtype=np.int32)
    n = _load().lso_hrw_topk(N, ctypes.c_uint64(key & 0xFFFFFFFFFFFFFFFF), K, _ptr(out))
    return out[:n]


def heuristic(alg, m, c, theta=0.0, k=0.0, tau=0.0) -> int:
    m = _c(m, np.float32); c = _c(c, np.float64)
    return int(_load().lso_heuristic(int(alg), m.shape[0], _ptr(m), _ptr(c), float(theta), float(k), float(tau)))


def policy(heuristic=1, count_cols=(-1, -1), theta_imbal=0.0, overload_k=0.0, prefix_tau=0.0, n_samples=0,
           n_min=0, lo=None, hi=None, epsilon=0.0, kv_col=-1, tau_sat=0.0, tau_ben=0.0, k_filter=0, delta=-1.0):
    """Policy parameters as the fp32 values the library receives (kept alive with the returned pair)."""
    f = lambda v: float(np.float32(v))
    lo_a = None if lo is None else _c(lo, np.float32)
    hi_a = None if hi is None else _c(hi, np.float32)
    p = Policy(int(heuristic), int(count_cols[0]), int(count_cols[1]), int(kv_col), int(k_filter), 0,
               f(theta_imbal), f(overload_k), f(prefix_tau), int(n_samples), int(n_min),
               f(epsilon), f(tau_sat), f(tau_ben), f(delta),
               None if lo_a is None else lo_a.ctypes.data, None if hi_a is None else hi_a.ctypes.data)
    return p, (lo_a, hi_a)


def route(mode, d, hidden, params, mu, inv_sigma, req_off, req_hashes, prompt_len, inst_feat, inst_off,
          inst_hashes, pol, rnd, sel=None, threads=0):
    """Alg. 3 + Alg. 4 decisions for the selected requests: (chosen, status, heuristic choice)."""
    lib = _load()
    hidden_a = _c(hidden, np.int32)
    params = _c(params, np.float32); mu = _c(mu, np.float32); inv_sigma = _c(inv_sigma, np.float32)
    req_off = _c(req_off, np.int64); req_hashes = _c(req_hashes, np.uint64)
    prompt_len = _c(prompt_len, np.int32); inst_feat = _c(inst_feat, np.float32)
    inst_off = _c(inst_off, np.int64); inst_hashes = _c(inst_hashes, np.uint64)
    rnd = _c(rnd, np.uint32)
    R = req_off.shape[0] - 1
    N = inst_off.shape[0] - 1
    sel_a = None if sel is None else _c(sel, np.int32)
    n_sel = R if sel_a is None else sel_a.shape[0]
    chosen = np.zeros(n_sel, np.int32); status = np.zeros(n_sel, np.int32); heur = np.zeros(n_sel, np.int32)
    p, _keep = pol
    rc = lib.lso_route(_mode(mode), d, hidden_a.shape[0], _ptr(hidden_a), _ptr(params), _ptr(mu), _ptr(inv_sigma),
                       n_sel, _ptr(sel_a), _ptr(req_off), _ptr(req_hashes), _ptr(prompt_len), N, _ptr(inst_feat),
                       _ptr(inst_off), _ptr(inst_hashes), ctypes.byref(p), _ptr(rnd), _ptr(chosen), _ptr(status),
                       _ptr(heur), threads)
    assert rc == 0, rc
    return chosen, status, heur


def embed(mode, d, hidden, params, mu, inv_sigma, x, y) -> np.ndarray:
    """Gradient-coreset embeddings (t - y) a_L of raw rows, [n x h_last] double."""
    lib = _load()
    h = _c(hidden, np.int32)
    x = _c(x, np.float32).reshape(-1, d); y = _c(y, np.float32)
    out = np.zeros((x.shape[0], int(h[-1])), np.float64)
    rc = lib.lso_embed(_mode(mode), d, h.shape[0], _ptr(h), _ptr(_c(params, np.float32)), _ptr(_c(mu, np.float32)),
                       _ptr(_c(inv_sigma, np.float32)), x.shape[0], _ptr(x), _ptr(y), _ptr(out))
    assert rc == 0, rc
    return out


class Buffer:
    """Host state of the two-pool training buffer (FIFO ring + replay pool)."""

    def __init__(self, d, fifo_cap, rep_cap):
        self.d, self.fifo_cap, self.rep_cap = d, fifo_cap, rep_cap
        self.fifo_count = np.zeros(1, np.int32); self.fifo_head = np.zeros(1, np.int32)
        self.fifo_x = np.zeros((fifo_cap, d), np.float32); self.fifo_y = np.zeros(fifo_cap, np.float32)
        self.rep_count = np.zeros(1, np.int32)
        self.rep_x = np.zeros((max(rep_cap, 1), d), np.float32); self.rep_y = np.zeros(max(rep_cap, 1), np.float32)

    def fifo_rows(self):
        idx = [(int(self.fifo_head[0]) + k) % self.fifo_cap for k in range(int(self.fifo_count[0]))]
        return self.fifo_x[idx], self.fifo_y[idx]

    def replay_rows(self):
        n = int(self.rep_count[0])
        return self.rep_x[:n], self.rep_y[:n]


def buffer_push(mode, hidden, params, mu, inv_sigma, buf, x, y) -> int:
    """Push rows into the buffer (FIFO, then gradient-coreset admission); returns the number admitted."""
    lib = _load()
    h = _c(hidden, np.int32)
    x = _c(x, np.float32).reshape(-1, buf.d); y = _c(y, np.float32)
    adm = np.zeros(1, np.int32)
    rc = lib.lso_buffer_push(_mode(mode), buf.d, h.shape[0], _ptr(h), _ptr(_c(params, np.float32)),
                             _ptr(_c(mu, np.float32)), _ptr(_c(inv_sigma, np.float32)), buf.fifo_cap, buf.rep_cap,
                             _ptr(buf.fifo_count), _ptr(buf.fifo_head), _ptr(buf.fifo_x), _ptr(buf.fifo_y),
                             _ptr(buf.rep_count), _ptr(buf.rep_x), _ptr(buf.rep_y), x.shape[0], _ptr(x), _ptr(y),
                             _ptr(adm))
    assert rc == 0, rc
    return int(adm[0])


def train_round(mode, hidden, params, mu, inv_sigma, buf, epochs, batch, lr, perm=None, dropout=None):
    """One retraining round over FIFO and pool; returns (new params, mean loss of the last epoch).
    dropout: None, or (p, seed, first step) -- minibatch u of the round is update call first step + u."""
    lib = _load()
    h = _c(hidden, np.int32)
    p = _c(params, np.float32).copy()
    perm_a = None if perm is None else _c(perm, np.int32)
    loss = np.zeros(1, np.float64)
    dp, seed, step0 = dropout if dropout is not None else (0.0, 0, 0)
    rc = lib.lso_train_round_dropout(_mode(mode), buf.d, h.shape[0], _ptr(h), _ptr(p), _ptr(_c(mu, np.float32)),
                                     _ptr(_c(inv_sigma, np.float32)), buf.fifo_cap, int(buf.fifo_count[0]),
                                     int(buf.fifo_head[0]), _ptr(buf.fifo_x), _ptr(buf.fifo_y), int(buf.rep_count[0]),
                                     _ptr(buf.rep_x), _ptr(buf.rep_y), int(epochs), int(batch), float(lr),
                                     _ptr(perm_a), float(dp), ctypes.c_uint64(seed), ctypes.c_uint64(step0),
                                     _ptr(loss))
    assert rc == 0, rc
    return p, float(loss[0])


# ---------------------------------------------------------------------------
# prefix-index maintenance (Section 2 / Section 4.2): exact LRU commit
# ---------------------------------------------------------------------------
def stamp(epoch: int, r: int, k: int) -> int:
    """Recency stamp of block k of request r committed in epoch `epoch`."""
    return int(_load().lso_stamp(epoch, r, k))


def initial_stamps(inst_off) -> np.ndarray:
    """Stamps of a loaded state: entry j of each instance's list gets j + 1."""
    inst_off = np.asarray(inst_off, np.int64)
    counts = np.diff(inst_off)
    out = np.empty(int(inst_off[-1]), np.uint64)
    for i, c in enumerate(counts):
        out[inst_off[i]:inst_off[i + 1]] = np.arange(1, c + 1, dtype=np.uint64)
    return out


def commit(inst_off, inst_hashes, inst_stamps, capacity, req_off, req_hashes, chosen, epoch):
    """One commit of a routed batch.  Returns (off, hashes, stamps) of the new
    lists, each instance's newest first."""
    inst_off = _c(inst_off, np.int64)
    N = len(inst_off) - 1
    cap = _c(capacity, np.int64)
    assert len(cap) == N
    req_off = _c(req_off, np.int64)
    R = len(req_off) - 1
    chosen = _c(chosen, np.int32)
    ih, ist = _c(inst_hashes, np.uint64), _c(inst_stamps, np.uint64)
    rh = _c(req_hashes, np.uint64)
    out_off = np.zeros(N + 1, np.int64)
    total = max(int(cap.sum()), 1)
    out_h = np.zeros(total, np.uint64)
    out_s = np.zeros(total, np.uint64)
    rc = _load().lso_commit(N, _ptr(inst_off), _ptr(ih), _ptr(ist), _ptr(cap), R, _ptr(req_off), _ptr(rh),
                            _ptr(chosen), epoch, _ptr(out_off), _ptr(out_h), _ptr(out_s))
    if rc:
        raise ValueError("commit arguments outside the stamp layout")
    n = int(out_off[-1])
    return out_off, out_h[:n].copy(), out_s[:n].copy()
