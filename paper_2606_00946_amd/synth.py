"""Seeded synthetic workloads for the batched routing scorer.

This module only draws inputs: prompts as block-hash lists, per-instance cached
block-hash sets, instance state rows, a randomly initialised reward model with
its normalisation statistics, and logged (features, TTFT) rows for the online
update.  It computes none of the scorer's own results (no prefix matching, no
normalisation, no MLP, no argmin), so the CPU oracle and the HIP path can both
take their inputs from here without sharing any of the method's arithmetic.

The paper evaluates on Mooncake traces and on synthetic prefix-sharing
workloads built from published KV-cache statistics (Section 5.1, Workloads);
neither is available here.  The recipes below stand in for them, with the
shapes the evaluation describes: prefix groups whose requests share a fixed
fraction of their prompt (10/30/50/70 %), Zipf group popularity, log-normal
prompt lengths, 16-token KV blocks, and per-instance caches filled by replaying
earlier requests under LRU.  Instance features follow the list in Section 4.1
(Features): running and queued requests, in-flight prefill and decode tokens,
KV-cache utilisation and a categorical accelerator class.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

BLOCK_TOKENS = 16
DERIVED_COLS = 5          # prompt_len, n_blocks, overlap, hit ratio, uncached tokens
MASK64 = np.uint64(0xFFFFFFFFFFFFFFFF)

# Stream tags keep chain, batch and warm-up hashes disjoint.
_CHAIN_TAG = 1 << 50
_BATCH_TAG = 1 << 51
_WARM_TAG = 1 << 52

_PREFIX_RATIOS = (0.1, 0.3, 0.5, 0.7)


@dataclasses.dataclass(frozen=True)
class WorkloadConfig:
    name: str
    seed: int
    R: int                      # requests in the scoring batch
    N: int                      # candidate instances
    groups: int                 # prefix groups
    zipf: float                 # group popularity exponent
    length: str                 # "fixed", "lognormal", "long"
    len_params: tuple           # distribution parameters (see _draw_lengths)
    capacity: tuple             # cached blocks per instance (per accelerator class)
    warmup_requests: int        # fixed replay count (0: replay until capacity)
    d: int                      # feature columns
    hidden: tuple               # hidden widths
    dtype: str                  # "fp32" or "bf16"
    update_batch: int           # online-update minibatch
    n_classes: int = 1          # accelerator classes (one-hot when > 1)
    lr: float = 1e-3

    @property
    def d_inst(self) -> int:
        return self.d - DERIVED_COLS

    @property
    def pairs(self) -> int:
        return self.R * self.N


CONFIGS = {
    "tiny": WorkloadConfig(
        name="tiny", seed=1001, R=64, N=8, groups=8, zipf=1.1,
        length="fixed", len_params=(512,), capacity=(2000,), warmup_requests=200,
        d=16, hidden=(64, 64), dtype="fp32", update_batch=256),
    "homogeneous": WorkloadConfig(
        name="homogeneous", seed=1002, R=4096, N=32, groups=64, zipf=1.0,
        length="lognormal", len_params=(7.0, 1.0, 64, 8192), capacity=(50_000,),
        warmup_requests=0, d=32, hidden=(128, 128), dtype="fp32", update_batch=4096),
    "heterogeneous": WorkloadConfig(
        name="heterogeneous", seed=1003, R=8192, N=64, groups=64, zipf=1.0,
        length="lognormal", len_params=(7.5, 1.2, 64, 16384),
        capacity=(100_000, 200_000, 400_000), warmup_requests=0, d=48,
        hidden=(256, 256), dtype="fp32", update_batch=8192, n_classes=3),
    "long_context": WorkloadConfig(
        name="long_context", seed=1004, R=2048, N=64, groups=16, zipf=0.8,
        length="long", len_params=(2048, 8192), capacity=(400_000,),
        warmup_requests=0, d=32, hidden=(128, 128), dtype="fp32", update_batch=4096),
    "large_batch": WorkloadConfig(
        name="large_batch", seed=1005, R=65536, N=256, groups=256, zipf=1.0,
        length="lognormal", len_params=(7.0, 1.0, 64, 8192), capacity=(100_000,),
        warmup_requests=0, d=64, hidden=(256, 256), dtype="bf16", update_batch=65536),
}


@dataclasses.dataclass
class Workload:
    cfg: WorkloadConfig
    # scoring batch (CSR over requests)
    req_off: np.ndarray         # int64 [R+1]
    req_hashes: np.ndarray      # uint64 [req_off[R]]
    prompt_len: np.ndarray      # int32 [R] tokens
    req_group: np.ndarray       # int32 [R] (generator bookkeeping only)
    # cache state (CSR over instances)
    inst_off: np.ndarray        # int64 [N+1]
    inst_hashes: np.ndarray     # uint64 [inst_off[N]]
    inst_feat: np.ndarray       # float32 [N, d_inst]
    # reward model
    params: np.ndarray          # float32 flat: per layer W [out, in] row-major then b [out]
    mu: np.ndarray              # float32 [d]
    inv_sigma: np.ndarray       # float32 [d]
    # online update samples
    upd_feats: np.ndarray       # float32 [B, d] raw feature rows
    upd_ttft: np.ndarray        # float32 [B] seconds
    lr: float


def layer_shapes(d: int, hidden) -> list:
    """(out, in) of every layer: d -> hidden[0] -> ... -> 1."""
    dims = [d, *hidden, 1]
    return [(dims[i + 1], dims[i]) for i in range(len(dims) - 1)]


def param_count(d: int, hidden) -> int:
    return sum(o * i + o for o, i in layer_shapes(d, hidden))


# --------------------------------------------------------------------------
# hashing used only to manufacture block ids
# --------------------------------------------------------------------------
def mix64(stream, pos) -> np.ndarray:
    """splitmix64 finaliser over (stream, position); the generator's block-id hash."""
    with np.errstate(over="ignore"):
        z = (np.asarray(stream, dtype=np.uint64) * np.uint64(0x9E3779B97F4A7C15)
             + (np.asarray(pos, dtype=np.uint64) + np.uint64(1)) * np.uint64(0xD1B54A32D192ED03))
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        z = z ^ (z >> np.uint64(31))
    return z


def _zipf_probs(G: int, a: float) -> np.ndarray:
    w = 1.0 / np.arange(1, G + 1, dtype=np.float64) ** a
    return w / w.sum()


def _draw_lengths(cfg: WorkloadConfig, rng, count: int):
    """Prompt lengths in tokens and their block counts."""
    if cfg.length == "fixed":
        L = np.full(count, cfg.len_params[0], dtype=np.int64)
    elif cfg.length == "lognormal":
        mu, sigma, lo, hi = cfg.len_params
        L = np.clip(np.rint(rng.lognormal(mu, sigma, count)), lo, hi).astype(np.int64)
    elif cfg.length == "long":
        nlo, nhi = cfg.len_params
        n = rng.integers(nlo, nhi + 1, count)
        L = n * BLOCK_TOKENS + rng.integers(0, BLOCK_TOKENS, count)
    else:
        raise ValueError(cfg.length)
    return L, L // BLOCK_TOKENS


def _shared_prefix(cfg: WorkloadConfig, rng, groups, n):
    """Blocks each request shares with its group's canonical chain."""
    if cfg.length == "long":
        q = rng.integers(8, 65, n.shape[0])          # private question suffix
        return np.maximum(n - q, 0)
    ratio = np.asarray(_PREFIX_RATIOS)[groups % len(_PREFIX_RATIOS)]
    return np.floor(ratio * n).astype(np.int64)


def _request_hashes(groups, n, s, ids):
    """Concatenated block hashes: chain[g][0:s) then private[id][s:n)."""
    total = int(n.sum())
    owner = np.repeat(np.arange(n.shape[0]), n)
    starts = np.concatenate([[0], np.cumsum(n)[:-1]])
    pos = np.arange(total, dtype=np.int64) - starts[owner]
    shared = pos < s[owner]
    stream = np.where(shared, _CHAIN_TAG + groups[owner], ids[owner]).astype(np.uint64)
    return mix64(stream, pos.astype(np.uint64))


# --------------------------------------------------------------------------
# cache state: replay warm-up requests, touch blocks tail-first, keep the
# C most recently used distinct blocks (LRU with capacity C)
# --------------------------------------------------------------------------
def _instance_cache(cfg: WorkloadConfig, rng, inst: int, capacity: int) -> np.ndarray:
    G = cfg.groups
    probs = _zipf_probs(G, cfg.zipf)
    offset = (inst * G) // cfg.N                # instance-specific group popularity
    warm_id_base = _WARM_TAG + (inst << 24)

    def draw(count):
        g = (rng.choice(G, size=count, p=probs) + offset) % G
        _, n = _draw_lengths(cfg, rng, count)
        s = _shared_prefix(cfg, rng, g, n)
        return g.astype(np.int64), n.astype(np.int64), s.astype(np.int64)

    if cfg.warmup_requests:
        g, n, s = draw(cfg.warmup_requests)
    else:
        g = np.zeros(0, np.int64); n = g.copy(); s = g.copy()
        mean_private = None
        while True:
            if mean_private is None:
                chunk = 256
            else:
                need = capacity - distinct
                chunk = int(max(64, 1.25 * need / max(mean_private, 1.0)))
            g2, n2, s2 = draw(chunk)
            g = np.concatenate([g, g2]); n = np.concatenate([n, n2]); s = np.concatenate([s, s2])
            priv = int((n - s).sum())
            chain = 0
            for grp in np.unique(g):
                chain += int(s[g == grp].max())
            distinct = priv + chain
            mean_private = priv / g.shape[0]
            if distinct >= capacity:
                break

    W = g.shape[0]
    tmax = np.int64(int(n.max()) + 1)
    w_idx = np.arange(W, dtype=np.int64)

    # private blocks: touched once, tail-first within their request
    pn = n - s
    p_owner = np.repeat(w_idx, pn)
    p_start = np.concatenate([[0], np.cumsum(pn)[:-1]])
    p_pos = (np.arange(int(pn.sum()), dtype=np.int64) - p_start[p_owner]) + s[p_owner]
    p_time = p_owner * tmax + (n[p_owner] - 1 - p_pos)

    # chain blocks: last touched by the latest warm-up of the group covering them
    c_grp, c_pos, c_time = [], [], []
    for grp in np.unique(g):
        sel = np.nonzero((g == grp) & (s > 0))[0]
        if sel.size == 0:
            continue
        smax = int(s[sel].max())
        last = np.full(smax, -1, dtype=np.int64)
        np.maximum.at(last, s[sel] - 1, sel)
        last = np.maximum.accumulate(last[::-1])[::-1]
        pos = np.arange(smax, dtype=np.int64)
        c_grp.append(np.full(smax, grp, dtype=np.int64))
        c_pos.append(pos)
        c_time.append(last * tmax + (n[last] - 1 - pos))
    c_grp = np.concatenate(c_grp) if c_grp else np.zeros(0, np.int64)
    c_pos = np.concatenate(c_pos) if c_pos else np.zeros(0, np.int64)
    c_time = np.concatenate(c_time) if c_time else np.zeros(0, np.int64)

    times = np.concatenate([p_time, c_time])
    keep = min(capacity, times.shape[0])
    order = np.argpartition(-times, keep - 1)[:keep] if keep < times.shape[0] else np.arange(times.shape[0])
    n_priv = p_time.shape[0]
    is_priv = order < n_priv
    pi = order[is_priv]
    ci = order[~is_priv] - n_priv
    priv_hash = mix64(np.uint64(warm_id_base) + p_owner[pi].astype(np.uint64), p_pos[pi].astype(np.uint64))
    chain_hash = mix64((_CHAIN_TAG + c_grp[ci]).astype(np.uint64), c_pos[ci].astype(np.uint64))
    hashes = np.concatenate([priv_hash, chain_hash])
    rng.shuffle(hashes)
    return hashes


def _instance_features(cfg: WorkloadConfig, rng, count: int, classes=None) -> np.ndarray:
    f = np.empty((count, cfg.d_inst), dtype=np.float64)
    f[:, 0] = rng.poisson(4.0, count)                 # queued requests
    f[:, 1] = rng.poisson(8.0, count)                 # running requests
    f[:, 2] = rng.uniform(0, 32768, count)            # in-flight prefill tokens
    f[:, 3] = rng.uniform(0, 32768, count)            # in-flight decode tokens
    f[:, 4] = rng.uniform(0, 1, count)                # KV-cache utilisation
    col = 5
    if cfg.n_classes > 1:
        if classes is None:
            classes = rng.integers(0, cfg.n_classes, count)
        f[:, col:col + cfg.n_classes] = 0.0
        f[np.arange(count), col + classes] = 1.0      # accelerator class, one-hot
        col += cfg.n_classes
    f[:, col:] = rng.uniform(0, 1, (count, cfg.d_inst - col))
    return f.astype(np.float32)


def _model(cfg: WorkloadConfig, rng) -> np.ndarray:
    """He-normal weights, small uniform biases, flat fp32."""
    parts = []
    for out_f, in_f in layer_shapes(cfg.d, cfg.hidden):
        parts.append(rng.normal(0.0, math.sqrt(2.0 / in_f), (out_f, in_f)).ravel())
        parts.append(rng.uniform(-0.1, 0.1, out_f))
    return np.concatenate(parts).astype(np.float32)


def _update_rows(cfg: WorkloadConfig, rng):
    """Logged (features, TTFT) rows: instance state, request length and a
    synthetic overlap for the pair, plus TTFT = linear(features) + log-normal noise."""
    B = cfg.update_batch
    inst = _instance_features(cfg, rng, B)
    L, n = _draw_lengths(cfg, rng, B)
    ov = np.minimum(np.floor(rng.uniform(0, 1, B) ** 2 * (n + 1)), n).astype(np.int64)
    rows = np.empty((B, cfg.d), dtype=np.float32)
    rows[:, :cfg.d_inst] = inst
    rows[:, cfg.d_inst + 0] = L
    rows[:, cfg.d_inst + 1] = n
    rows[:, cfg.d_inst + 2] = ov
    rows[:, cfg.d_inst + 3] = (BLOCK_TOKENS * ov) / np.maximum(L, 1)
    rows[:, cfg.d_inst + 4] = L - BLOCK_TOKENS * ov
    x = rows.astype(np.float64)
    mean = x.mean(axis=0)
    std = x.std(axis=0)
    std[std == 0] = 1.0
    a = rng.normal(0.0, 1.0 / math.sqrt(cfg.d), cfg.d)
    y = np.maximum(0.01, ((x - mean) / std) @ a + 0.5) + rng.lognormal(math.log(0.05), 0.5, B)
    return rows, y.astype(np.float32), mean, std


def generate(name_or_cfg, *, R: int | None = None, N: int | None = None) -> Workload:
    """Build the seeded workload; R/N overrides shrink a config for quick tests."""
    cfg = CONFIGS[name_or_cfg] if isinstance(name_or_cfg, str) else name_or_cfg
    if R is not None or N is not None:
        cfg = dataclasses.replace(cfg, R=R or cfg.R, N=N or cfg.N)
    ss = np.random.SeedSequence(cfg.seed)
    s_req, s_inst, s_feat, s_model, s_upd = ss.spawn(5)

    # scoring batch
    rng = np.random.Generator(np.random.PCG64(s_req))
    groups = rng.choice(cfg.groups, size=cfg.R, p=_zipf_probs(cfg.groups, cfg.zipf)).astype(np.int64)
    L, n = _draw_lengths(cfg, rng, cfg.R)
    s = _shared_prefix(cfg, rng, groups, n)
    ids = _BATCH_TAG + np.arange(cfg.R, dtype=np.int64)
    req_hashes = _request_hashes(groups, n, s, ids)
    req_off = np.zeros(cfg.R + 1, dtype=np.int64)
    np.cumsum(n, out=req_off[1:])

    # cache state
    classes = np.arange(cfg.N) % cfg.n_classes
    inst_streams = s_inst.spawn(cfg.N)
    lists = []
    for i in range(cfg.N):
        cap = cfg.capacity[classes[i] % len(cfg.capacity)]
        lists.append(_instance_cache(cfg, np.random.Generator(np.random.PCG64(inst_streams[i])), i, cap))
    inst_off = np.zeros(cfg.N + 1, dtype=np.int64)
    np.cumsum([x.shape[0] for x in lists], out=inst_off[1:])
    inst_hashes = np.concatenate(lists) if lists else np.zeros(0, np.uint64)

    rng = np.random.Generator(np.random.PCG64(s_feat))
    inst_feat = _instance_features(cfg, rng, cfg.N, classes if cfg.n_classes > 1 else None)

    params = _model(cfg, np.random.Generator(np.random.PCG64(s_model)))
    rows, y, mean, std = _update_rows(cfg, np.random.Generator(np.random.PCG64(s_upd)))

    return Workload(
        cfg=cfg, req_off=req_off, req_hashes=req_hashes.astype(np.uint64),
        prompt_len=L.astype(np.int32), req_group=groups.astype(np.int32),
        inst_off=inst_off, inst_hashes=inst_hashes.astype(np.uint64), inst_feat=inst_feat,
        params=params, mu=mean.astype(np.float32), inv_sigma=(1.0 / std).astype(np.float32),
        upd_feats=rows, upd_ttft=y, lr=cfg.lr)
