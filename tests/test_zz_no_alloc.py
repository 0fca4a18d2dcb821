"""emb_cache_forward_noalloc (the forward with the library's static scratch instead of the
workspace) against emb_cache_forward, through the C ABI: pooled outputs bit for bit and
the forward statistics equal, on two calls in a row, the second with a smaller input,
and a call beyond the scratch's size refused without enqueueing anything."""
import ctypes

import numpy as np
import pytest

from common import custom_cfg
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


def _cfg():
    return custom_cfg(rows=[3000, 777, 20000], dim=64, bits=4, sb_fp16=True, cache_fraction=0.05, assoc=8,
                      batch=256, pooling=("poisson", 12), rounding="stochastic", optimizer="adagrad")


def test_forward_noalloc_matches_forward(torch):
    from paper_2010_11305_amd.emb_cache import EmbCache

    cfg = _cfg()
    T, d = len(cfg["rows"]), cfg["dim"]
    print("forward_noalloc: 3 tables, d64 INT4, two calls (256 then 97 bags)", flush=True)
    g = EmbCache(cfg, max_indices=20000)
    g.init_uniform(cfg["init_lo"], cfg["init_hi"], cfg["init_seed"])
    # two training steps first, so that lookups hit the cache and miss it
    for k in range(2):
        st = workload.make_step(cfg, k)
        idx = torch.from_numpy(st["indices"]).cuda()
        off = torch.from_numpy(st["offsets"]).cuda()
        g.forward(idx, off, cfg["batch"])
        g.backward_update(idx, off, cfg["batch"], torch.from_numpy(st["grad"]).cuda())
    for k, B in ((2, 256), (3, 97)):
        c = dict(cfg, batch=B)
        idx_np, off_np = workload.make_indices(c, k)
        idx = torch.from_numpy(idx_np).cuda()
        off = torch.from_numpy(off_np).cuda()
        ref = g.forward(idx, off, B)
        torch.cuda.synchronize()
        ref_stats = [g.stats(t) for t in range(T)]
        out = torch.full((B, T, d), float("nan"), dtype=torch.float32, device="cuda")
        g.forward_noalloc(idx, off, B, out)
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy().view(np.uint32), ref.cpu().numpy().view(np.uint32)), (k, B)
        assert [g.stats(t) for t in range(T)] == ref_stats
        assert ref_stats[2]["hit_lookups"] > 0 and ref_stats[2]["hit_lookups"] < ref_stats[2]["lookups"]
    assert g.check() == 0


def test_forward_noalloc_refuses_more_than_its_scratch(torch):
    from paper_2010_11305_amd import emb_cache as ec

    cfg = _cfg()
    g = ec.EmbCache(cfg, max_indices=20000)
    L = ec.load()
    fake = ctypes.c_void_p(1 << 20)   # never dereferenced: the size check comes first
    limit = (64 << 20) // 4 - 64
    st = L.emb_cache_forward_noalloc(g._h, fake, limit + 1, fake, 4, fake, None)
    assert st == ec.EMB_ENOMEM
    assert g.check() == 0
