"""GPU parity at the full sizes of the industrial and stress workloads, in the launch
configuration the benchmark times (all tables in one call).

* industrial (100 x 5M x d128 INT4): 32 steps, into the steady regime of evictions the
  benchmark times; table 0 against the oracle bit for bit (pooled outputs and statistics
  every step, the whole table state twice); sampled tables against the invariants that
  hold at any size.
* stress (1 x 200M x d256 INT8): the oracle cannot initialise 200M rows in a test, so
  the full-size run is checked by invariants and by exact sums of sampled bags from
  the exported rows; a row-scaled slice (2M rows, same shape otherwise) runs against
  the oracle bit for bit.
"""
import numpy as np
import pytest

from common import oracle_from_cfg
from exact import dequant_exact
from parity import assert_f32, assert_same, compare_state, log
from paper_2010_11305_amd import configs, workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2010_11305_amd import emb_cache
    emb_cache.load()
    return t


def check_invariants(g, cfg, t, st):
    c = g.export_cache(t)
    tags = c["tag"]
    valid = tags >= 0
    A, ns = cfg["assoc"], g.n_sets[t]
    assert len(np.unique(tags[valid])) == valid.sum(), f"duplicate tags t{t}"
    assert np.all(tags[valid] % ns == np.nonzero(valid)[0] // A), f"tag in the wrong set t{t}"
    if cfg["policy"] == "lru":
        assert np.all((c["ts"] >= 0) == valid) and np.all(c["ts"][valid] < g.step)
    assert np.all(np.isfinite(c["crow"][valid]))
    s = g.stats(t)
    assert s["inserts"] + s["bypasses"] == s["unique"] - s["unique_hits"]
    assert s["evictions"] == s["inserts"] - s["empty_fills"]
    assert s["bwd_lookups"] == st


def bag_sums(g, cfg, t, idx, off, bags):
    """Exact left-to-right sums of sampled bags from the exported state of table t."""
    c = g.export_cache(t)
    where = {int(r): k for k, r in enumerate(c["tag"]) if r >= 0}
    out = []
    for b in bags:
        rows = idx[off[b]:off[b + 1]]
        acc = np.zeros(cfg["dim"], dtype=np.float32)
        for i, r in enumerate(rows):
            r = int(r)
            if r in where:
                x = c["crow"][where[r]]
            else:
                e = g.export_rows(t, r, 1)
                x = dequant_exact(e["codes"][0], e["scale"][0], e["bias"][0])
            acc = x.copy() if i == 0 else (acc + x).astype(np.float32)
        out.append(acc)
    return np.array(out)


def test_industrial_full_size_table0_and_invariants(torch):
    """32 steps in the benchmark's launch configuration (4 input batches cycled, gradients
    drawn on the GPU), so that the cache reaches the steady regime the benchmark times:
    table 0 bit for bit against the oracle (pooled outputs and statistics every step, the
    whole table state at steps 15 and 31), sampled tables against the invariants."""
    from paper_2010_11305_amd.emb_cache import EmbCache
    cfg = configs.get("industrial")
    T, B, d = len(cfg["rows"]), cfg["batch"], cfg["dim"]
    pool = [workload.make_indices(cfg, k) for k in range(4)]
    log("industrial: 4 input batches ready, GPU state 36.6 GB")
    g = EmbCache(cfg, max_indices=max(p[0].size for p in pool))
    g.init_uniform(cfg["init_lo"], cfg["init_hi"], cfg["init_seed"])
    one = configs.get("industrial", rows=[cfg["rows"][0]])
    o = oracle_from_cfg(one)
    log("industrial: oracle init of table 0 (5M rows)")
    o.init_uniform(cfg["init_lo"], cfg["init_hi"], cfg["init_seed"])
    gen = torch.Generator(device="cuda")
    gen.manual_seed(cfg["grad_seed"])
    dev = [(torch.from_numpy(i).cuda(), torch.from_numpy(f).cuda()) for i, f in pool]
    evicted = 0
    for k in range(32):
        idx_np, off_np = pool[k % 4]
        idx, off = dev[k % 4]
        grad = torch.randn((B, T, d), generator=gen, device="cuda", dtype=torch.float32) * cfg["grad_sigma"]
        out = g.forward(idx, off, B).cpu().numpy()
        n0 = int(off_np[B])
        ref = o.forward(idx_np[:n0], off_np[:B + 1], B)
        assert_f32(out[:, 0:1], ref, f"industrial step {k} pooled table 0")
        g.backward_update(idx, off, B, grad)
        o.backward_update(idx_np[:n0], off_np[:B + 1], B, np.ascontiguousarray(grad[:, 0:1].cpu().numpy()))
        assert g.stats(0) == o.stats(0), (g.stats(0), o.stats(0))
        evicted += g.stats(0)["evictions"]
        if k % 8 == 7:
            lens = np.diff(off_np).reshape(T, B).sum(axis=1)
            for t in (0, 1, 37, 63, 99):
                check_invariants(g, cfg, t, int(lens[t]))
        if k in (15, 31):
            compare_state(o, g, one)
        log(f"industrial step {k}: table 0 matches ({g.stats(0)['evictions']} evictions)")
    assert evicted > 32 * 20000   # the steady regime: tens of thousands of evictions per step in table 0
    assert g.check() == 0


def test_stress_full_size_properties(torch):
    from paper_2010_11305_amd.emb_cache import EmbCache
    cfg = configs.get("stress")
    B = cfg["batch"]
    log("stress: 200M rows x d256 INT8 (52.8 GB)")
    st0 = workload.make_step(cfg, 0)
    g = EmbCache(cfg, max_indices=st0["indices"].size + 64)
    g.init_uniform(cfg["init_lo"], cfg["init_hi"], cfg["init_seed"])
    rng = np.random.default_rng(7)
    for k in range(3):
        st = st0 if k == 0 else workload.make_step(cfg, k)
        idx = torch.from_numpy(st["indices"]).cuda()
        off = torch.from_numpy(st["offsets"]).cuda()
        bags = rng.choice(B, size=24, replace=False)
        want = bag_sums(g, cfg, 0, st["indices"], st["offsets"], bags)
        out = g.forward(idx, off, B).cpu().numpy()
        assert_f32(out[bags, 0], want, f"stress step {k} sampled bags")
        g.backward_update(idx, off, B, torch.from_numpy(st["grad"]).cuda())
        check_invariants(g, cfg, 0, int(st["indices"].size))
        # rows written this step: every code in range, scale/bias finite
        rows = np.unique(st["indices"])[:: max(1, st["indices"].size // 5000)]
        for r in rows[:200]:
            e = g.export_rows(0, int(r), 1)
            assert np.isfinite(e["scale"][0]) and np.isfinite(e["bias"][0]) and e["scale"][0] >= 0
        log(f"stress step {k}: sampled bags exact, invariants hold")
    assert g.check() == 0


def test_stress_row_slice_parity(torch):
    from paper_2010_11305_amd.emb_cache import EmbCache
    cfg = configs.get("stress", rows=[2_000_000], batch=4096)
    log("stress slice: 2M rows x d256 INT8, 32-way LRU, SR")
    o = oracle_from_cfg(cfg)
    o.init_uniform(cfg["init_lo"], cfg["init_hi"], cfg["init_seed"])
    st = [workload.make_step(cfg, k) for k in range(4)]
    g = EmbCache(cfg, max_indices=max(s["indices"].size for s in st))
    g.init_uniform(cfg["init_lo"], cfg["init_hi"], cfg["init_seed"])
    from parity import step_both
    for s in st:
        step_both(o, g, cfg, s, torch)
    compare_state(o, g, cfg)
