"""Helpers for the GPU tests: upload a workload, run the HIP path through the C
ABI, bring results back, and compare against the oracle."""
from __future__ import annotations

import sys

import numpy as np

from paper_2606_00946_amd import lodestar


def note(msg: str) -> None:
    """Name the case before a GPU step, flushed, so a failing run says where it was."""
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def to_dev(a):
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint64:
        a = a.view(np.int64)
    return torch.from_numpy(a).to("cuda")


BAND_REL = 2.0 ** -7           # half-width of the candidate band, relative to sum_j |w3_j| h2_j + |b3|


def uses_fast_path(d, hidden, dtype, exact=False):
    """Whether a context scores on the bf16 matrix-core path (mirrors the library's rule)."""
    return (dtype == "bf16" and not exact and d in (16, 32, 48, 64) and len(hidden) == 2
            and hidden[0] == hidden[1] and hidden[0] in (64, 128, 256))


def bf16_np(x):
    """Round float32 values to bf16 (ties to even), vectorised; finite inputs."""
    u = np.ascontiguousarray(x, np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def head_magnitude(w, rows):
    """sum_j |w3_j| h2_j + |b3| for raw feature rows, bf16 model (the scale of the band)."""
    d, (h1, h2) = w.cfg.d, w.cfg.hidden
    p = w.params
    o = 0
    W1 = p[o:o + h1 * d].reshape(h1, d); o += h1 * d
    b1 = p[o:o + h1]; o += h1
    W2 = p[o:o + h2 * h1].reshape(h2, h1); o += h2 * h1
    b2 = p[o:o + h2]; o += h2
    W3 = p[o:o + h2]; o += h2
    b3 = p[o]
    xt = bf16_np(((rows.astype(np.float32) - w.mu) * w.inv_sigma).astype(np.float32)).astype(np.float64)
    a1 = bf16_np(np.maximum(xt @ bf16_np(W1).astype(np.float64).T + b1, 0).astype(np.float32)).astype(np.float64)
    a2 = bf16_np(np.maximum(a1 @ bf16_np(W2).astype(np.float64).T + b2, 0).astype(np.float32)).astype(np.float64)
    return a2 @ np.abs(bf16_np(W3).astype(np.float64)) + abs(float(b3))


class GpuRun:
    """A context loaded with one workload's model and cache state."""

    def __init__(self, w, dtype=None, params=None, exact=False, prefix_join=0, prefix_closed=False):
        import torch
        self.w = w
        cfg = w.cfg
        self.ctx = lodestar.Context(cfg.d, cfg.hidden, dtype or cfg.dtype)
        self.exact = exact
        if exact:
            self.ctx.ls_set_exact_scores(True)
        if prefix_join:
            self.ctx.ls_set_prefix_join(prefix_join)
        if prefix_closed:
            self.ctx.ls_set_prefix_closed(True)
        self.ctx.ls_set_model(w.params if params is None else params, w.mu, w.inv_sigma)
        self.inst_hashes = to_dev(w.inst_hashes)
        self.ctx.ls_load_cache_state(w.inst_off, self.inst_hashes)
        self.req_off = to_dev(w.req_off)
        self.req_hashes = to_dev(w.req_hashes)
        self.prompt_len = to_dev(w.prompt_len.astype(np.int32))
        self.inst_feat = to_dev(w.inst_feat.astype(np.float32))
        torch.cuda.synchronize()

    def score(self, with_optional=True):
        import torch
        R, N, d = self.w.cfg.R, self.w.cfg.N, self.w.cfg.d
        out = {
            "chosen": torch.full((R,), -7, dtype=torch.int32, device="cuda"),
            "min_ttft": torch.zeros(R, dtype=torch.float32, device="cuda") if with_optional else None,
            "scores": torch.zeros(R * N, dtype=torch.float32, device="cuda") if with_optional else None,
            "overlap": torch.full((R * N,), -7, dtype=torch.int32, device="cuda") if with_optional else None,
            "feat": torch.zeros(R * d, dtype=torch.float32, device="cuda") if with_optional else None,
        }
        self.ctx.ls_score_batch(self.req_off, self.req_hashes, self.prompt_len, self.inst_feat, out["chosen"],
                                out["min_ttft"], out["scores"], out["overlap"], out["feat"])
        torch.cuda.synchronize()
        res = {k: (v.cpu().numpy() if v is not None else None) for k, v in out.items()}
        if with_optional:
            res["scores"] = res["scores"].reshape(R, N)
            res["overlap"] = res["overlap"].reshape(R, N)
            res["feat"] = res["feat"].reshape(R, d)
        return res

    def update(self, feats=None, ttft=None, lr=None):
        import torch
        w = self.w
        feats = w.upd_feats if feats is None else feats
        ttft = w.upd_ttft if ttft is None else ttft
        lr = w.lr if lr is None else lr
        loss = torch.zeros(1, dtype=torch.float32, device="cuda")
        grad = torch.zeros(self.ctx.n_params, dtype=torch.float32, device="cuda")
        self.ctx.ls_update(to_dev(np.asarray(feats, np.float32)), to_dev(np.asarray(ttft, np.float32)), lr, loss, grad)
        torch.cuda.synchronize()
        params, _, _ = self.ctx.ls_get_model()
        return {"loss": float(loss.cpu().numpy()[0]), "grad": grad.cpu().numpy(), "params": params}


def rel_ok(got, ref, rtol=1e-4, floor=0.1):
    """Elementwise |got - ref| <= rtol * max(|ref|, floor * rms(ref)).

    A value that nearly cancels cannot carry 1e-4 relative accuracy in any fixed
    precision, so its error is measured against a fraction of its tensor's scale."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return True, 0.0
    rms = float(np.sqrt(np.mean(ref * ref)))
    scale = np.maximum(np.abs(ref), floor * rms)
    scale[scale == 0] = 1e-30
    err = np.abs(got - ref) / scale
    return bool(np.all(err <= rtol)), float(err.max())


def layer_slices(d, hidden):
    dims = [d, *hidden, 1]
    out, off = [], 0
    for i in range(len(dims) - 1):
        n = dims[i] * dims[i + 1]
        out.append((f"W{i + 1}", off, off + n)); off += n
        out.append((f"b{i + 1}", off, off + dims[i + 1])); off += dims[i + 1]
    return out
