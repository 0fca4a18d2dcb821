"""Input generator checks: Zipf sampler against the exact pmf, the rank->row map
is a bijection, offsets/shape contracts of every named config."""
import numpy as np
import pytest

from paper_2010_11305_amd import configs, workload


@pytest.mark.parametrize("N,alpha", [(50, 1.1), (20, 0.5), (20, 2.0), (1000, 1.05), (7, 1.0)])
def test_zipf_sampler_matches_pmf(N, alpha):
    s = workload.ZipfSampler(N, alpha).sample(np.random.default_rng(N), 400_000)
    assert s.min() >= 1 and s.max() <= N
    k = np.arange(1, N + 1)
    p = k ** -alpha
    p /= p.sum()
    obs = np.bincount(s, minlength=N + 1)[1:]
    chi2 = ((obs - p * s.size) ** 2 / (p * s.size)).sum()
    dof = N - 1
    assert chi2 < dof + 6 * np.sqrt(2 * dof)


@pytest.mark.parametrize("N", [1, 2, 97, 1000, 5_000_000])
def test_affine_map_is_bijection(N):
    a, c = workload.affine_bijection(3, 5, N)
    if N <= 100_000:
        rows = (a * np.arange(N, dtype=np.int64) + c) % N
        assert np.array_equal(np.sort(rows), np.arange(N))
    assert np.gcd(a, N) == 1


@pytest.mark.parametrize("name", ["tiny", "kaggle_int8", "kaggle_int4"])
def test_step_shapes(name):
    cfg = configs.get(name)
    st = workload.make_step(cfg, 0)
    T, B = len(cfg["rows"]), cfg["batch"]
    off = st["offsets"]
    assert off.dtype == np.int32 and off.size == T * B + 1 and off[0] == 0 and np.all(np.diff(off) >= 0)
    assert st["indices"].size == off[-1]
    for t in range(T):
        seg = st["indices"][off[t * B]:off[(t + 1) * B]]
        assert seg.min() >= 0 and seg.max() < cfg["rows"][t]
    assert st["grad"].shape == (B, T, cfg["dim"]) and st["grad"].dtype == np.float32
    again = workload.make_step(cfg, 0)
    assert np.array_equal(again["indices"], st["indices"])


def test_industrial_single_table_slice():
    cfg = configs.get("industrial")
    idx, off = workload.make_indices(cfg, 0, tables=[3])
    B = cfg["batch"]
    assert off[3 * B] == 0 and off[4 * B] == idx.size and off[-1] == idx.size
    L = idx.size
    assert 0.9 * 30 * B < L < 1.1 * 30 * B
    u, c = np.unique(idx, return_counts=True)
    assert 0.05 < c.max() / L < 0.4          # Zipf 1.2 top row takes a large share


def test_drift_moves_the_hot_rows_between_phases():
    """With drift (period P, fraction f), the hottest rows are the same within a phase
    and move by f*N row ids (through the bijection) at a phase boundary."""
    cfg = configs.get("tiny", rows=[10000], batch=4096, pooling=("fixed", 1), zipf=1.2, drift=(5, 0.25))
    top = []
    for k in (0, 4, 5, 9, 10):
        idx, _ = workload.make_indices(cfg, k)
        v, c = np.unique(idx, return_counts=True)
        top.append(set(v[np.argsort(-c)[:20]].tolist()))
    assert len(top[0] & top[1]) >= 15 and len(top[2] & top[3]) >= 15      # same phase
    assert len(top[0] & top[2]) <= 2 and len(top[2] & top[4]) <= 2        # next phase
    # the hottest rank maps to a + c' mod N with c' moved by 2500 per phase
    a, c = workload.affine_bijection(cfg["index_seed"], 0, 10000)
    assert {c % 10000, (c + 2500) % 10000, (c + 5000) % 10000} <= top[0] | top[2] | top[4]
    # without drift the stream is unchanged
    base = configs.get("tiny", rows=[10000], batch=4096, pooling=("fixed", 1), zipf=1.2)
    assert np.array_equal(workload.make_indices(base, 3)[0], workload.make_indices(dict(base, drift=None), 3)[0])
