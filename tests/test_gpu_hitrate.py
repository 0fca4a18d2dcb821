"""GPU checks behind the synthetic hit-rate study (paper_2010_11305_amd.hitrate):
the library's statistics equal the oracle's on a drifting stream, step by step, for
each policy of the study, and the hit rate grows with the cache."""
import numpy as np
import pytest

from common import custom_cfg
from parity import compare_state, log, make_pair, step_both
from paper_2010_11305_amd import workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2010_11305_amd import emb_cache
    emb_cache.load()
    return t


@pytest.mark.parametrize("policy,assoc,decay", [("lru", 32, 0), ("lfu", 32, 0), ("lfu", 32, 5), ("lru", 1, 0),
                                                ("lfu", 1, 0)])
def test_drift_stream_matches_oracle(torch, policy, assoc, decay):
    cfg = custom_cfg(rows=[5000], batch=512, pooling=("fixed", 1), zipf=1.05, drift=(4, 0.37),
                     cache_fraction=0.05, assoc=assoc, policy=policy, lfu_decay_interval=decay)
    log(f"drift stream {policy} assoc={assoc} decay={decay}")
    o, g = make_pair(cfg)
    for k in range(12):
        step_both(o, g, cfg, workload.make_step(cfg, k), torch)
    compare_state(o, g, cfg)


def test_hit_rate_grows_with_cache(torch):
    from paper_2010_11305_amd import hitrate
    cfg, steps = hitrate.stream("stationary", 8)
    cfg = dict(cfg, rows=[100_000], batch=4096)
    steps = [workload.make_indices(cfg, k) for k in range(8)]
    log("hit rate vs cache size")
    rates = [hitrate.hit_rate(dict(cfg, cache_fraction=f, assoc=32, policy="lfu"), steps, 4)
             for f in (0.01, 0.05, 0.2)]
    assert 0 < rates[0] < rates[1] < rates[2] < 1, rates
