"""GPU parity: the HIP library (through the C ABI) against the CPU oracle, same
seeded inputs, every state array compared after every step (see parity.py)."""
import numpy as np
import pytest

from common import custom_cfg, oracle_from_cfg
from parity import assert_f32, assert_same, compare_state, log, make_pair, step_both, to_dev
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


INIT_CASES = ([(d, b, sb) for d in (16, 32, 64, 128, 256) for b in (8, 4, 2) for sb in (False, True)]
              + [(d, 16, False) for d in (16, 32, 64, 128, 256)])


@pytest.mark.parametrize("dim,bits,sb16", INIT_CASES)
def test_init_uniform_parity(torch, dim, bits, sb16):
    cfg = custom_cfg(rows=[1000, 37, 2049], dim=dim, bits=bits, sb_fp16=sb16)
    log(f"init parity dim={dim} bits={bits} sb16={sb16}")
    o, g = make_pair(cfg)
    compare_state(o, g, cfg)


@pytest.mark.parametrize("over", [{}, {"bits": 16, "rounding": "stochastic"}, {"bits": 2, "sb_fp16": True}])
def test_forward_from_imported_state(torch, over):
    """Oracle trains 4 steps; its state is imported into the GPU; pooled outputs match."""
    cfg = custom_cfg(**over)
    log(f"forward from imported oracle state {over}")
    o, g = make_pair(cfg)
    for k in range(4):
        st = workload.make_step(cfg, k)
        o.forward(st["indices"], st["offsets"], st["batch"])
        o.backward_update(st["indices"], st["offsets"], st["batch"], st["grad"])
    r, c = o.export_rows(0), o.export_cache(0)
    g.import_rows(0, 0, r["codes"], r["scale"], r["bias"], r["cnt"], r["G"])
    g.import_cache(0, c["crow"], c["tag"], c["ts"])
    g.step = o.step
    compare_state(o, g, cfg)
    st = workload.make_step(cfg, 4)
    idx, off, _ = to_dev(st, torch)
    out_g = g.forward(idx, off, st["batch"]).cpu().numpy()
    out_o = o.forward(st["indices"], st["offsets"], st["batch"])
    assert_f32(out_g, out_o, "pooled")
    assert g.stats(0)["hit_lookups"] == o.stats(0)["hit_lookups"] > 0


STEP_CASES = {
    "tiny": {},
    "tiny_sr": {"rounding": "stochastic"},
    "tiny_int4_fp16_lfu_adagrad": {"bits": 4, "sb_fp16": True, "policy": "lfu", "lfu_decay_interval": 3,
                                   "rounding": "stochastic", "optimizer": "adagrad"},
    "tiny_assoc1_lru": {"assoc": 1, "cache_fraction": 0.05},
    "tiny_assoc1_lfu": {"assoc": 1, "policy": "lfu"},
    "tiny_assoc2_lfu_sgd": {"assoc": 2, "policy": "lfu", "cache_fraction": 0.1},
    "tiny_assoc32_bigcache": {"assoc": 32, "cache_fraction": 0.3, "batch": 300, "pooling": ("uniform", 1, 12)},
    "tiny_nocache": {"cache_fraction": 0.0},
    "tiny_fullcover": {"cache_fraction": 1.024, "assoc": 32},
    "d32_int4": {"dim": 32, "bits": 4, "rounding": "stochastic"},
    "d64_int8_adagrad": {"dim": 64, "optimizer": "adagrad"},
    "d128_int4_fp16_lru16": {"dim": 128, "bits": 4, "sb_fp16": True, "assoc": 16, "cache_fraction": 0.05,
                             "rounding": "stochastic", "optimizer": "adagrad", "pooling": ("poisson", 30), "zipf": 1.2},
    "d256_int8_sr": {"dim": 256, "rounding": "stochastic", "assoc": 32, "cache_fraction": 0.1, "lr": 0.05},
    "hot_row": {"rows": [300], "zipf": 2.0, "batch": 600, "pooling": ("uniform", 1, 8), "assoc": 8},
    "assoc64": {"assoc": 64, "cache_fraction": 0.3, "batch": 300, "pooling": ("uniform", 1, 12)},
    "fp16_rne": {"bits": 16},
    "fp16_sr_lfu_adagrad": {"bits": 16, "rounding": "stochastic", "policy": "lfu", "optimizer": "adagrad",
                            "lfu_decay_interval": 3},
    "fp16_direct_mapped_lfu": {"bits": 16, "assoc": 1, "policy": "lfu", "rounding": "stochastic"},
    "d128_fp16_sr_lru16": {"dim": 128, "bits": 16, "rounding": "stochastic", "assoc": 16, "cache_fraction": 0.05,
                           "pooling": ("poisson", 30), "zipf": 1.2},
    "int2_rne": {"bits": 2},
    "d64_int2_fp16sb_sr_adagrad": {"dim": 64, "bits": 2, "sb_fp16": True, "rounding": "stochastic",
                                   "optimizer": "adagrad"},
    "d256_int2_sr_assoc32": {"dim": 256, "bits": 2, "rounding": "stochastic", "assoc": 32, "cache_fraction": 0.1},
    "int2_nocache_sr": {"bits": 2, "cache_fraction": 0.0, "rounding": "stochastic"},
    "multi_table": {"rows": [1000, 5, 64, 3000], "batch": 96, "assoc": 4, "cache_fraction": 0.05},
    "odd_tables": {"rows": [1, 2, 3, 7, 97, 641, 1001, 4093, 5000, 65537, 100003, 2], "batch": 200, "assoc": 8,
                   "cache_fraction": 0.07, "pooling": ("uniform", 1, 6)},
    "odd_tables_lfu_dm": {"rows": [3, 17, 999, 12289, 3], "batch": 150, "assoc": 1, "policy": "lfu",
                          "cache_fraction": 0.3},
    # tables whose key ranges fit 16 bits while their sum needs 18: the per-table sort
    # (2 digit passes per segment, several tiles per table, a 5-row table in one tile)
    "seg_tables": {"rows": [40000, 5, 60001, 300, 50000, 30000], "batch": 512, "assoc": 8, "cache_fraction": 0.05,
                   "pooling": ("poisson", 12), "zipf": 1.1},
    "seg_tables_lfu_sr_adagrad": {"rows": [40000, 5, 60001, 300, 50000, 30000], "batch": 512, "assoc": 4,
                                  "cache_fraction": 0.02, "policy": "lfu", "rounding": "stochastic",
                                  "optimizer": "adagrad", "bits": 4, "sb_fp16": True, "dim": 32,
                                  "pooling": ("poisson", 12), "zipf": 1.1},
    # rows with more than 512 lookups at every row width: bag blocks of 32768/d bags, staged
    # in halves, with ragged last blocks and halves (d32: 1500 bags = blocks of 1024; d64:
    # 700 of 512; d256: 300 of 128)
    "big_rows_d32": {"rows": [200, 3000], "dim": 32, "batch": 1500, "pooling": ("poisson", 6), "zipf": 1.5,
                     "assoc": 8, "cache_fraction": 0.1},
    "big_rows_d64_lfu_sr": {"rows": [150, 900], "dim": 64, "batch": 700, "pooling": ("poisson", 5), "zipf": 1.4,
                            "assoc": 4, "cache_fraction": 0.05, "policy": "lfu", "rounding": "stochastic",
                            "bits": 4, "sb_fp16": True},
    "big_rows_d256_adagrad": {"rows": [120], "dim": 256, "batch": 300, "pooling": ("poisson", 8), "zipf": 1.3,
                              "assoc": 16, "cache_fraction": 0.3, "optimizer": "adagrad", "rounding": "stochastic"},
    "big_rows_d128_fp16": {"rows": [400, 77], "dim": 128, "batch": 520, "pooling": ("poisson", 4), "zipf": 1.6,
                           "assoc": 2, "cache_fraction": 0.05, "bits": 16, "optimizer": "adagrad"},
    # 360 small tables: every segment's keys fit one digit pass, their sum needs two
    "seg_tables_small": {"rows": [200, 250, 17, 240, 1, 199] * 60, "batch": 40, "assoc": 2, "cache_fraction": 0.05,
                         "pooling": ("uniform", 0, 5)},
}


def sort_passes(cfg):
    """Digit passes of the sort of the whole key, and of the per-table sort (the
    library picks the latter when it takes fewer passes)."""
    ranges = []
    for n in cfg["rows"]:
        sets = int(np.floor(cfg["cache_fraction"] * n)) // cfg["assoc"] if cfg["cache_fraction"] > 0 else 0
        if cfg["cache_fraction"] > 0:
            sets = max(sets, 1)
        ranges.append(sets * -(-n // sets) if sets else n)
    total = sum(ranges)
    return (int(total).bit_length() + 7) // 8, (int(max(ranges)).bit_length() + 7) // 8


@pytest.mark.parametrize("case", list(STEP_CASES))
def test_step_parity(torch, case):
    cfg = custom_cfg(**STEP_CASES[case])
    log(f"step parity {case}: rows={cfg['rows'][:4]} dim={cfg['dim']} bits={cfg['bits']} assoc={cfg['assoc']}")
    o, g = make_pair(cfg)
    for k in range(8):
        st = workload.make_step(cfg, k)
        step_both(o, g, cfg, st, torch)
        compare_state(o, g, cfg)
    s = o.stats(0)
    if cfg["cache_fraction"] > 0:
        assert s["inserts"] + s["unique_hits"] > 0


# Rows of 128 and 256 columns are handled with split columns per lane (columns [4g, 4g+4)
# and [d/2+4g, d/2+4g+4)), their codes loaded and stored in place in the row update and
# the eviction, and INT8 codes read with their (scale, bias) in one load in the gather:
# every code width and (scale, bias) format at both widths, with stochastic rounding and
# row-wise Adagrad, under LRU (inserts and bypasses), direct-mapped LRU and LFU (residents
# updated and then displaced).
WIDE_POLICIES = {"lru": {"policy": "lru", "assoc": 4}, "direct": {"policy": "lru", "assoc": 1},
                 "lfu": {"policy": "lfu", "assoc": 4, "lfu_decay_interval": 2}}
WIDE_CASES = [(d, b, sb, pol) for d in (128, 256) for (b, sb) in ((8, False), (8, True), (4, False), (4, True),
                                                                    (2, False), (2, True), (16, False))
              for pol in WIDE_POLICIES]


@pytest.mark.parametrize("dim,bits,sb16,policy", WIDE_CASES)
def test_wide_row_layouts(torch, dim, bits, sb16, policy):
    cfg = custom_cfg(rows=[600, 37], dim=dim, bits=bits, sb_fp16=sb16, cache_fraction=0.05, rounding="stochastic",
                     optimizer="adagrad", lr=0.05, batch=96, pooling=("uniform", 1, 5), zipf=1.2,
                     **WIDE_POLICIES[policy])
    log(f"wide rows dim={dim} bits={bits} sb16={sb16} policy={policy}")
    o, g = make_pair(cfg)
    tot = {"inserts": 0, "bypasses": 0, "hit_evictions": 0}
    for k in range(6):
        st = workload.make_step(cfg, k)
        step_both(o, g, cfg, st, torch)
        compare_state(o, g, cfg)
        s = o.stats(0)
        for n in tot:
            tot[n] += s[n]
    assert tot["inserts"] > 0 and tot["bypasses"] > 0
    if policy != "lru":
        assert tot["hit_evictions"] > 0


@pytest.mark.parametrize("case", ["multi_table", "seg_tables_lfu_sr_adagrad", "big_rows_d64_lfu_sr"])
def test_tables_without_lookups(torch, case):
    """Steps in which some tables (first, last, in the middle, all but one) have only
    empty bags: their unique-row ranges are empty, their sort segments hold no key, and
    the other tables still match the oracle bit for bit, statistics included."""
    cfg = custom_cfg(**STEP_CASES[case])
    T = len(cfg["rows"])
    subsets = [[t for t in range(T) if t not in (1, T - 2)] or [0], [0], [T - 1], list(range(1, T - 1)) or [0],
               [t for t in range(T) if t % 2 == 1] or [0], list(range(T))]
    log(f"tables without lookups {case}: T={T} subsets={subsets}")
    o, g = make_pair(cfg)
    for k, sub in enumerate(subsets):
        st = workload.make_step(cfg, k, tables=sub)
        step_both(o, g, cfg, st, torch)
        compare_state(o, g, cfg)
        for t in range(T):
            if t not in sub:
                assert g.stats(t)["unique"] == 0


HOST_TABLE_CASES = ["tiny", "tiny_int4_fp16_lfu_adagrad", "fp16_sr_lfu_adagrad", "d128_int4_fp16_lru16",
                    "tiny_nocache", "d64_int2_fp16sb_sr_adagrad"]


@pytest.mark.parametrize("case", HOST_TABLE_CASES)
def test_step_parity_host_table(torch, case):
    """The low-precision table in pinned host memory (reached over the host link), the
    cache in device memory: the same bits as the oracle."""
    cfg = custom_cfg(**STEP_CASES[case])
    log(f"host-table step parity {case}")
    o, g = make_pair(cfg, table="host")
    assert g.table is not None and g.table.is_pinned()
    for k in range(6):
        step_both(o, g, cfg, workload.make_step(cfg, k), torch)
        compare_state(o, g, cfg)


def _bags_of(rows, per_bag, rng):
    rows = np.array(rows, dtype=np.int32)
    rng.shuffle(rows)
    B = (len(rows) + per_bag - 1) // per_bag
    off = np.minimum(np.arange(B + 1) * per_bag, len(rows)).astype(np.int32)
    return rows, off, B


@pytest.mark.parametrize("dim", [16, 128])
def test_lfu_hot_rows_displaced_after_update(torch, dim):
    """LFU, one set of 2 ways holding rows 1 and 2.  Next step row 1 is hit 70 times
    while rows 3 and 4 miss 100 and 90 times: row 3 displaces row 2 (not accessed),
    row 4 displaces row 1 after row 1's own update; rows 1, 3, 4 have > 64 lookups,
    so their merged gradients come from chunk sums."""
    cfg = custom_cfg(rows=[64], cache_fraction=2 / 64, assoc=2, policy="lfu", optimizer="adagrad",
                     rounding="stochastic", bits=4, sb_fp16=True, dim=dim, lr=0.05)
    log(f"LFU hot-row hit eviction, dim={dim}")
    o, g = make_pair(cfg, max_indices=1024)
    assert o.n_sets == [1] and g.n_sets == [1]
    rng = np.random.default_rng(dim)
    for rows in ([1, 2], [1] * 70 + [3] * 100 + [4] * 90 + [5, 6, 7]):
        idx, off, B = _bags_of(rows, 4, rng)
        grad = (rng.standard_normal((B, 1, dim)) * 0.1).astype(np.float32)
        step_both(o, g, cfg, {"indices": idx, "offsets": off, "batch": B, "grad": grad}, torch)
        compare_state(o, g, cfg)
    s = o.stats(0)
    assert s["hit_evictions"] == 1 and s["inserts"] == 2 and s["evictions"] == 2
    assert sorted(o.export_cache(0)["tag"].tolist()) == [3, 4]


def test_kaggle_int8_full_size(torch):
    """26 Table-1 tables at full size: 12 steps, outputs every step, whole state at the end."""
    cfg = configs.get("kaggle_int8")
    log("kaggle_int8 full size: oracle init (33.7M rows) ...")
    o, g = make_pair(cfg)
    for k in range(12):
        step_both(o, g, cfg, workload.make_step(cfg, k), torch)
    log("kaggle_int8: comparing state")
    compare_state(o, g, cfg)


def test_kaggle_int4_full_size(torch):
    """12 steps (across the LFU decay at step 10); LFU displaces residents right after
    their own update here (hit evictions), which the state comparison covers."""
    cfg = configs.get("kaggle_int4")
    log("kaggle_int4 full size: oracle init (33.7M rows) ...")
    o, g = make_pair(cfg)
    hit_evictions = 0
    for k in range(12):   # crosses the LFU decay at step 10
        step_both(o, g, cfg, workload.make_step(cfg, k), torch)
        hit_evictions += sum(g.stats(t)["hit_evictions"] for t in range(len(cfg["rows"])))
    log(f"kaggle_int4: comparing state ({hit_evictions} hit evictions)")
    assert hit_evictions > 0
    compare_state(o, g, cfg)


def test_big_row_cases_have_rows_past_512_lookups():
    """The cases above reach the block sums (a row with more than 512 lookups in a step)."""
    for case in ("big_rows_d32", "big_rows_d64_lfu_sr", "big_rows_d256_adagrad", "big_rows_d128_fp16"):
        cfg = custom_cfg(**STEP_CASES[case])
        idx, off = workload.make_indices(cfg, 0)
        B = cfg["batch"]
        most = max(np.bincount(idx[off[t * B]:off[(t + 1) * B]]).max() for t in range(len(cfg["rows"])))
        assert most > 512, case


def test_seg_cases_take_the_per_table_sort():
    for case in ("seg_tables", "seg_tables_lfu_sr_adagrad", "seg_tables_small"):
        whole, seg = sort_passes(custom_cfg(**STEP_CASES[case]))
        assert seg < whole, case
    whole, seg = sort_passes(configs.get("industrial"))
    assert (whole, seg) == (4, 3)


def test_per_table_sort_with_skipped_lookups(torch):
    """Per-table sort with skipped lookups inside bags (negative and out-of-range rows),
    positions before the first and after the last bag, and tables without lookups."""
    from paper_2010_11305_amd.emb_cache import EMB_EINDEX
    cfg = custom_cfg(**dict(STEP_CASES["seg_tables"], batch=64))
    assert sort_passes(cfg)[1] < sort_passes(cfg)[0]
    rng = np.random.default_rng(11)
    T, B = len(cfg["rows"]), cfg["batch"]
    o, g = make_pair(cfg, max_indices=8192)
    for k in range(4):
        idx, off = [int(v) for v in rng.integers(-3, 10, size=3)], [3]
        for t in range(T):
            n_t = cfg["rows"][t]
            for b in range(B):
                m = 0 if (t == 3 or (t == 1 and k % 2)) else int(rng.integers(0, 9))
                r = np.minimum(rng.zipf(1.2, size=m) - 1, n_t - 1)
                bad = rng.random(m) < 0.1
                r[bad] = rng.choice([-1, n_t, n_t + 7, -(2 ** 31)], size=int(bad.sum()))
                idx += [int(v) for v in r]
                off.append(len(idx))
        idx += [5, -1]
        st = {"indices": np.array(idx, dtype=np.int32), "offsets": np.array(off, dtype=np.int32), "batch": B,
              "grad": rng.standard_normal((B, T, cfg["dim"])).astype(np.float32)}
        log(f"per-table sort with skipped lookups: step {k}, {len(idx)} positions")
        step_both(o, g, cfg, st, torch)
        compare_state(o, g, cfg)
        assert g.check() == EMB_EINDEX


def test_invalid_indices_and_empty_bags(torch):
    from paper_2010_11305_amd.emb_cache import EMB_EINDEX, EMB_OK
    cfg = custom_cfg(batch=4)
    log("invalid indices / empty bags")
    o, g = make_pair(cfg, max_indices=64)
    st = {"indices": np.array([5, -1, 7, 1000, 3], dtype=np.int32), "offsets": np.array([0, 0, 2, 4, 5], dtype=np.int32),
          "batch": 4, "grad": np.ones((4, 1, 16), dtype=np.float32)}
    step_both(o, g, cfg, st, torch)
    compare_state(o, g, cfg)
    assert g.check() == EMB_EINDEX
    assert g.check() == EMB_OK


def test_malformed_offsets_skip_the_step(torch):
    from paper_2010_11305_amd.emb_cache import EMB_EINDEX
    cfg = custom_cfg(batch=4)
    log("malformed offsets")
    o, g = make_pair(cfg, max_indices=64)
    before = g.export_rows(0)
    idx = torch.tensor([1, 2, 3, 4, 5], dtype=torch.int32, device="cuda")
    off = torch.tensor([0, 3, 2, 5, 5], dtype=torch.int32, device="cuda")   # decreasing
    grad = torch.ones((4, 1, 16), dtype=torch.float32, device="cuda")
    g.forward(idx, off, 4)          # results unspecified, but no fault and the flag is set
    assert g.check() == EMB_EINDEX
    g.backward_update(idx, off, 4, grad)
    assert g.check() == EMB_EINDEX
    after = g.export_rows(0)
    assert np.array_equal(before["codes"], after["codes"]) and g.stats(0)["unique"] == 0


def test_malformed_offsets_per_table_sort(torch):
    """Malformed offsets with the per-table sort (every key skipped, the stream one
    segment): no fault, the flag set, no state change; the next good step matches the oracle."""
    from paper_2010_11305_amd.emb_cache import EMB_EINDEX, EMB_OK
    cfg = custom_cfg(**dict(STEP_CASES["seg_tables"], batch=64))
    assert sort_passes(cfg)[1] < sort_passes(cfg)[0]
    T, B = len(cfg["rows"]), cfg["batch"]
    log("malformed offsets, per-table sort")
    o, g = make_pair(cfg, max_indices=20000)
    st = workload.make_step(cfg, 0)
    before = [g.export_rows(t) for t in range(T)]
    off = st["offsets"].copy()
    off[T * B // 2] = off[-1] + 5   # past the end
    idx_t, _, grad_t = to_dev(st, torch)
    off_t = torch.from_numpy(off).cuda()
    g.backward_update(idx_t, off_t, B, grad_t)
    assert o.backward_update(st["indices"], off, B, st["grad"])   # the oracle rejects it too
    assert g.check() == EMB_EINDEX
    for t in range(T):
        assert np.array_equal(before[t]["codes"], g.export_rows(t)["codes"]) and g.stats(t)["unique"] == 0
    assert g.step == o.step == 1   # the rejected call still counts a step on both sides
    compare_state(o, g, cfg)
    step_both(o, g, cfg, workload.make_step(cfg, 1), torch)
    compare_state(o, g, cfg)
    assert g.check() == EMB_OK


def test_malformed_offsets_on_a_decay_step(torch):
    """LFU with counts halved every 2 steps: the call of step 2 (a decay step) has
    malformed offsets.  It is rejected on both sides without halving the counts, both
    count the step, and the next steps (3 without decay, 4 with) match the oracle."""
    from paper_2010_11305_amd.emb_cache import EMB_EINDEX, EMB_OK
    cfg = custom_cfg(policy="lfu", lfu_decay_interval=2, assoc=4, rounding="stochastic")
    B = cfg["batch"]
    log("malformed offsets on an LFU decay step")
    o, g = make_pair(cfg)
    for k in range(2):
        step_both(o, g, cfg, workload.make_step(cfg, k), torch)
    counts = g.export_rows(0)["cnt"].copy()
    assert counts.max() > 1
    st = workload.make_step(cfg, 2)
    off = st["offsets"].copy()
    off[B // 2] = -1
    idx_t, _, grad_t = to_dev(st, torch)
    g.backward_update(idx_t, torch.from_numpy(off).cuda(), B, grad_t)
    assert o.backward_update(st["indices"], off, B, st["grad"])
    assert g.check() == EMB_EINDEX
    assert np.array_equal(g.export_rows(0)["cnt"], counts)   # no decay on the rejected step
    assert g.step == o.step == 3
    compare_state(o, g, cfg)
    for k in (3, 4):
        step_both(o, g, cfg, workload.make_step(cfg, k), torch)
        compare_state(o, g, cfg)
    assert g.check() == EMB_OK


@pytest.mark.parametrize("case", ["tiny", "seg_tables"])
def test_empty_steps(torch, case):
    """A step without bags (B = 0) and a step whose bags are all empty (no lookups): no
    fault, no error, pooled outputs +0, no state change; the oracle agrees on both, and
    a full step afterwards still matches it."""
    from paper_2010_11305_amd.emb_cache import EMB_OK
    cfg = custom_cfg(**dict(STEP_CASES.get(case, {}), batch=32))
    T, B, d = len(cfg["rows"]), cfg["batch"], cfg["dim"]
    log(f"empty steps {case}")
    o, g = make_pair(cfg, max_indices=30000)
    step_both(o, g, cfg, workload.make_step(cfg, 0), torch)
    before = [g.export_rows(t) for t in range(T)]
    # no bags at all
    st0 = {"indices": np.zeros(0, dtype=np.int32), "offsets": np.zeros(1, dtype=np.int32), "batch": 0,
           "grad": np.zeros((0, T, d), dtype=np.float32)}
    step_both(o, g, cfg, st0, torch)
    # B bags per table, every one empty
    st1 = {"indices": np.zeros(0, dtype=np.int32), "offsets": np.zeros(T * B + 1, dtype=np.int32), "batch": B,
           "grad": np.ones((B, T, d), dtype=np.float32)}
    idx, off, grad = to_dev(st1, torch)
    out = g.forward(idx, off, B)
    assert not torch.any(out != 0) and not torch.any(torch.signbit(out))
    o.forward(st1["indices"], st1["offsets"], B)
    g.backward_update(idx, off, B, grad)
    o.backward_update(st1["indices"], st1["offsets"], B, st1["grad"])
    torch.cuda.synchronize()
    assert g.check() == EMB_OK
    for t in range(T):
        a = g.export_rows(t)
        assert np.array_equal(a["codes"], before[t]["codes"]) and g.stats(t) == o.stats(t)
    compare_state(o, g, cfg)
    step_both(o, g, cfg, workload.make_step(cfg, 1), torch)
    compare_state(o, g, cfg)


def test_determinism_and_resume(torch):
    cfg = custom_cfg(bits=4, sb_fp16=True, rounding="stochastic", policy="lfu", lfu_decay_interval=2,
                     optimizer="adagrad", assoc=4)
    log("determinism / resume")
    _, g1 = make_pair(cfg)
    _, g2 = make_pair(cfg)
    for k in range(3):
        for g in (g1, g2):
            st = workload.make_step(cfg, k)
            idx, off, grad = to_dev(st, torch)
            g.backward_update(idx, off, st["batch"], grad)
    r, c = g2.export_rows(0), g2.export_cache(0)
    _, g3 = make_pair(cfg)
    g3.import_rows(0, 0, r["codes"], r["scale"], r["bias"], r["cnt"], r["G"])
    g3.import_cache(0, c["crow"], c["tag"], c["ts"])
    g3.step = g2.step
    for k in range(3, 6):
        for g in (g1, g3):
            st = workload.make_step(cfg, k)
            idx, off, grad = to_dev(st, torch)
            g.backward_update(idx, off, st["batch"], grad)
    a, b = g1.export_rows(0), g3.export_rows(0)
    for key in a:
        assert np.array_equal(a[key], b[key]), key
    assert np.array_equal(g1.export_cache(0)["crow"], g3.export_cache(0)["crow"])


@pytest.mark.parametrize("policy", ["lru", "lfu"])
def test_adagrad_accumulators_follow_the_rows(torch, policy):
    """A row's Adagrad accumulator lives in its record while the row is not cached and in
    its cache slot's entry while it is.  Steps that insert and evict, then cache imports
    that empty the cache and fill it again on a handle that holds residents: the
    accumulators the rows export never change, and the next step still matches the
    oracle bit for bit."""
    cfg = custom_cfg(bits=4, sb_fp16=True, rounding="stochastic", policy=policy, optimizer="adagrad", assoc=4,
                     **({"lfu_decay_interval": 2} if policy == "lfu" else {}))
    log(f"accumulators follow the rows ({policy})")
    o, g = make_pair(cfg)
    for k in range(4):
        step_both(o, g, cfg, workload.make_step(cfg, k), torch)
    assert sum(g.stats(0)[f] for f in ("inserts", "evictions")) > 0
    compare_state(o, g, cfg)
    G0 = g.export_rows(0)["G"]
    assert np.count_nonzero(G0) > 0
    c = g.export_cache(0)
    cached = c["tag"] >= 0
    assert cached.sum() > 0 and np.count_nonzero(G0[c["tag"][cached]]) > 0
    g.import_cache(0, np.zeros_like(c["crow"]), np.full_like(c["tag"], -1), np.full_like(c["ts"], -1))
    assert np.array_equal(g.export_rows(0)["G"], G0)
    g.import_cache(0, c["crow"], c["tag"], c["ts"])
    assert np.array_equal(g.export_rows(0)["G"], G0)
    # a row's accumulator written while it is cached, read back, then moved out and in
    r = g.export_rows(0)
    G1 = G0.copy()
    G1[c["tag"][cached]] += 1.0
    g.import_rows(0, 0, r["codes"], r["scale"], r["bias"], r["cnt"], G1)
    assert np.array_equal(g.export_rows(0)["G"], G1)
    g.import_rows(0, 0, r["codes"], r["scale"], r["bias"], r["cnt"], G0)
    compare_state(o, g, cfg)
    step_both(o, g, cfg, workload.make_step(cfg, 4), torch)
    compare_state(o, g, cfg)


def test_update_timing_events(torch):
    """The measurement events around the row-update kernel: one duration per timed call,
    and timing does not change results."""
    cfg = custom_cfg(batch=64)
    log("update timing events")
    o, g = make_pair(cfg)
    g.set_update_timing(True)
    for k in range(3):
        step_both(o, g, cfg, workload.make_step(cfg, k), torch)
    ms = g.update_times(8)
    g.set_update_timing(False)
    assert ms.shape == (3,) and np.all(ms > 0) and np.all(ms < 1000)
    compare_state(o, g, cfg)
