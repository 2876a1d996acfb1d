"""Properties of the synthetic inputs that tests and options rely on."""
import numpy as np
import pytest

from paper_2606_00946_amd import synth


@pytest.mark.parametrize("name,k", [("tiny", 64), ("homogeneous", 200), ("large_batch", 60)])
def test_caches_are_prefix_closed(name, k):
    """Every replayed request touches its blocks tail-first under LRU, so a
    cached block's predecessors in any prompt are cached too: along every
    sampled prompt, the cached positions on every instance form a prefix."""
    w = synth.generate(name)
    rng = np.random.default_rng(1)
    sel = rng.choice(w.cfg.R, min(k, w.cfg.R), replace=False)
    sets = [set(w.inst_hashes[w.inst_off[i]:w.inst_off[i + 1]].tolist()) for i in range(w.cfg.N)]
    for r in sel:
        h = w.req_hashes[w.req_off[r]:w.req_off[r + 1]].tolist()
        for s in sets:
            cached = [x in s for x in h]
            first_miss = cached.index(False) if False in cached else len(cached)
            assert not any(cached[first_miss:]), (name, int(r))
