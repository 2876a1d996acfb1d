"""Prefix-index maintenance through the C ABI against the oracle (Section 2: the
gateway records routed prefixes, engines evict least recently used blocks).

After every commit each instance's list -- its blocks and their recency
stamps -- must equal the oracle's exactly, and overlaps computed on the
rebuilt tables must equal the oracle's overlaps on its lists."""
import numpy as np
import pytest

import oracle
from gpu_helpers import note, to_dev
from paper_2606_00946_amd import lodestar, synth

pytestmark = pytest.mark.gpu


def device_lists(ctx):
    off, h, st = ctx.ls_read_cache_state()
    return off, h.cpu().numpy().view(np.uint64), st.cpu().numpy().view(np.uint64)


def canonical(off, h, st):
    """Each instance's entries ordered by stamp (stamps are unique per instance)."""
    inst = np.repeat(np.arange(len(off) - 1), np.diff(off))
    order = np.lexsort((st, inst))
    return inst[order], h[order], st[order]


def assert_same_lists(dev, ref, tag):
    np.testing.assert_array_equal(dev[0], ref[0], err_msg=f"{tag}: list lengths")
    a, b = canonical(*dev), canonical(*ref)
    np.testing.assert_array_equal(a[1], b[1], err_msg=f"{tag}: blocks")
    np.testing.assert_array_equal(a[2], b[2], err_msg=f"{tag}: stamps")


def batch_slice(w, a, b):
    off = w.req_off[a:b + 1] - w.req_off[a]
    return off, w.req_hashes[w.req_off[a]:w.req_off[b]], w.prompt_len[a:b]


def make_ctx(w, capacity, inst_off=None, inst_hashes=None):
    cfg = w.cfg
    ctx = lodestar.Context(cfg.d, cfg.hidden, cfg.dtype)
    ctx.ls_set_model(w.params, w.mu, w.inv_sigma)
    ctx.ls_set_cache_capacity(capacity)
    io = w.inst_off if inst_off is None else inst_off
    ih = w.inst_hashes if inst_hashes is None else inst_hashes
    ctx.ls_load_cache_state(io, to_dev(ih))
    return ctx


def gpu_overlap(ctx, w, off, hashes, L):
    import torch
    R, N = len(off) - 1, ctx.n_instances
    chosen = torch.zeros(R, dtype=torch.int32, device="cuda")
    ov = torch.zeros(R * N, dtype=torch.int32, device="cuda")
    ctx.ls_score_batch(to_dev(off), to_dev(hashes), to_dev(L.astype(np.int32)),
                       to_dev(w.inst_feat.astype(np.float32)), chosen, overlap=ov)
    return chosen.cpu().numpy(), ov.cpu().numpy().reshape(R, N)


def test_commits_match_oracle():
    """Four commits in a row on the homogeneous workload (32 instances of 50,000
    blocks): capacities equal to, below, above the loaded size and 0; one batch
    routed by the scorer, the others at random with requests sent nowhere."""
    w = synth.generate("homogeneous", R=1024)
    N = w.cfg.N
    counts = np.diff(w.inst_off)
    cap = counts.copy()
    cap[1] = counts[1] // 2
    cap[2] = counts[2] + 5000
    cap[3] = 0
    cap[4] = 7
    ctx = make_ctx(w, cap)
    ref = (w.inst_off.copy(), w.inst_hashes.copy(), oracle.initial_stamps(w.inst_off))
    note("index: load under capacities")
    dev = device_lists(ctx)
    # the loaded lists are the loaded hashes (no duplicates in this workload), stamped by position
    assert_same_lists(dev, ref, "load")
    rng = np.random.default_rng(3)
    for epoch, (a, b) in enumerate([(0, 256), (256, 512), (512, 768), (768, 1024)], start=1):
        off, hashes, L = batch_slice(w, a, b)
        if epoch == 2:
            chosen, _ = gpu_overlap(ctx, w, off, hashes, L)
        else:
            chosen = rng.integers(-1, N + 1, b - a).astype(np.int32)
        note(f"index: commit {epoch}")
        ctx.ls_commit_routes(to_dev(off), to_dev(hashes), to_dev(chosen))
        ref = oracle.commit(*ref, cap, off, hashes, chosen, epoch)
        assert_same_lists(device_lists(ctx), ref, f"commit {epoch}")
    # the rebuilt tables answer overlaps on the committed state
    off, hashes, L = batch_slice(w, 0, 300)
    note("index: overlaps after the commits")
    _, ov = gpu_overlap(ctx, w, off, hashes, L)
    want = oracle.overlap(off, hashes, ref[0], ref[1])
    np.testing.assert_array_equal(ov, want)
    assert ov.max() > 0
    ctx.close()


def test_commit_edge_cases():
    """Hand-built state: repeated blocks in the loaded lists (the newest kept), the
    all-ones block hash, capacity 0, an empty commit, empty requests, repeated
    blocks within a request, a request longer than the capacity."""
    w = synth.generate("tiny")
    ones = 2**64 - 1
    lists = [[5, 6, 5, 7], [ones, 9, 10], [11, 12], [13]] + [[100 + i] for i in range(w.cfg.N - 4)]
    inst_off = np.zeros(len(lists) + 1, np.int64)
    inst_off[1:] = np.cumsum([len(x) for x in lists])
    inst_h = np.array([v for x in lists for v in x], np.uint64)
    N = len(lists)
    cap = np.array([3, 4, 0, 2] + [1] * (N - 4), np.int64)
    ctx = make_ctx(w, cap, inst_off, inst_h)
    # the oracle's view of the loaded state: repeated blocks keep their newest entry
    st0 = oracle.initial_stamps(inst_off)
    ref = oracle.commit(inst_off, inst_h, st0, np.diff(inst_off) + 10, np.zeros(1, np.int64),
                        np.zeros(0, np.uint64), np.zeros(0, np.int32), 1)
    ref = (ref[0], ref[1], ref[2])
    note("index edge: load with repeated blocks")
    assert_same_lists(device_lists(ctx), ref, "load")
    reqs = [[ones, 20, 21], [], [5, 5, 30], [40, 41, 42, 43, 44, 45], [9], [13, 50]]
    chosen = np.array([1, 0, 0, 3, 1, 3], np.int32)
    roff = np.zeros(len(reqs) + 1, np.int64)
    roff[1:] = np.cumsum([len(x) for x in reqs])
    rh = np.array([v for x in reqs for v in x], np.uint64)
    for epoch, (o, h, c) in enumerate([(roff, rh, chosen), (np.zeros(1, np.int64), np.zeros(0, np.uint64),
                                                          np.zeros(0, np.int32)), (roff, rh, chosen[::-1].copy())],
                                      start=1):
        note(f"index edge: commit {epoch}")
        import torch
        hd = to_dev(h) if h.size else torch.zeros(0, dtype=torch.int64, device="cuda")
        cd = to_dev(c) if c.size else torch.zeros(0, dtype=torch.int32, device="cuda")
        ctx.ls_commit_routes(to_dev(o), hd, cd)
        ref = oracle.commit(*ref, cap, o, h, c, epoch)
        assert_same_lists(device_lists(ctx), ref, f"edge commit {epoch}")
    ctx.close()


def test_commit_errors():
    w = synth.generate("tiny")
    cfg = w.cfg
    ctx = lodestar.Context(cfg.d, cfg.hidden, cfg.dtype)
    ctx.ls_set_model(w.params, w.mu, w.inv_sigma)
    ctx.ls_load_cache_state(w.inst_off, to_dev(w.inst_hashes))
    off, hashes, _ = batch_slice(w, 0, 4)
    note("index errors")
    with pytest.raises(lodestar.LodestarError) as e:            # loaded without capacities
        ctx.ls_commit_routes(to_dev(off), to_dev(hashes), to_dev(np.zeros(4, np.int32)))
    assert e.value.code == lodestar.LS_ERR_STATE
    with pytest.raises(lodestar.LodestarError) as e:
        ctx.ls_set_cache_capacity(np.full(cfg.N, -1, np.int64))
    assert e.value.code == lodestar.LS_ERR_INVALID
    ctx.close()


def test_commit_large_batch():
    """The Large batch (65,536 requests x 256 instances, 100,000 blocks each):
    route with the scorer, commit, compare every instance's list with the
    oracle; then overlaps of sampled requests on the committed tables."""
    w = synth.generate("large_batch")
    N = w.cfg.N
    cap = np.diff(w.inst_off)
    ctx = make_ctx(w, cap)
    note("index large: route")
    chosen, _ = gpu_overlap(ctx, w, w.req_off, w.req_hashes, w.prompt_len)
    note("index large: commit")
    ctx.ls_commit_routes(to_dev(w.req_off), to_dev(w.req_hashes), to_dev(chosen))
    ref = oracle.commit(w.inst_off, w.inst_hashes, oracle.initial_stamps(w.inst_off), cap, w.req_off, w.req_hashes,
                        chosen, 1)
    assert_same_lists(device_lists(ctx), ref, "large commit")
    sel = np.random.default_rng(9).choice(w.cfg.R, 64, replace=False)
    rows = [w.req_hashes[w.req_off[r]:w.req_off[r + 1]] for r in sel]
    off = np.zeros(len(sel) + 1, np.int64)
    off[1:] = np.cumsum([len(x) for x in rows])
    hashes = np.concatenate(rows)
    note("index large: overlaps after the commit")
    _, ov = gpu_overlap(ctx, w, off, hashes, w.prompt_len[sel])
    np.testing.assert_array_equal(ov, oracle.overlap(off, hashes, ref[0], ref[1]))
    # the last request routed to an instance holds the newest stamps there: its
    # whole prompt is cached on that instance after the commit
    last = {}
    for r, i in enumerate(chosen):
        last[int(i)] = r
    sel2 = np.array(sorted(last.values())[:64])
    rows = [w.req_hashes[w.req_off[r]:w.req_off[r + 1]] for r in sel2]
    off = np.zeros(len(sel2) + 1, np.int64)
    off[1:] = np.cumsum([len(x) for x in rows])
    note("index large: last requests of each instance")
    _, ov = gpu_overlap(ctx, w, off, np.concatenate(rows), w.prompt_len[sel2])
    np.testing.assert_array_equal(ov[np.arange(len(sel2)), chosen[sel2]], np.diff(off))
    ctx.close()
