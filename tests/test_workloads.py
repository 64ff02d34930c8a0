"""The seeded synthetic workloads: shapes, determinism, row independence and structure."""
import numpy as np
import pytest

from workloads import CONFIGS, generate


@pytest.mark.parametrize("name", list(CONFIGS))
def test_rows_are_reproducible_and_independent(name):
    cfg = CONFIGS[name]
    a = generate(name, rows=[0, 3, 5])
    b = generate(name, rows=[5, 3])
    assert a["p"].shape == (3, cfg.V) and a["p"].dtype == np.float32
    assert a["drafts"].shape == (3, cfg.K) and a["drafts"].dtype == np.int32
    assert np.array_equal(a["p"][2], b["p"][0]) and np.array_equal(a["q"][1], b["q"][1])
    assert np.array_equal(a["drafts"][2], b["drafts"][0]) and np.array_equal(a["u"][2], b["u"][0])
    # drafted tokens lie in the draft support; uniforms are 24-bit dyadics in [0, 1)
    for i in range(3):
        assert np.all(a["q"][i][a["drafts"][i]] > 0)
    k = a["u"].astype(np.float64) * (1 << 24)
    assert np.all(k == np.floor(k)) and np.all(a["u"] < 1) and np.all(a["u"] >= 0)
    # rows are probability vectors up to the fp32 cast
    assert np.allclose(a["p"].astype(np.float64).sum(1), 1, atol=1e-5)
    assert np.allclose(a["q"].astype(np.float64).sum(1), 1, atol=1e-5)


def test_topk_support():
    w = generate("k3top1024", rows=[0, 1])
    for i in range(2):
        assert np.count_nonzero(w["q"][i]) == 1024
        assert np.count_nonzero(w["p"][i]) == w["p"].shape[1]


def test_zipf_target_is_a_permuted_power_law():
    w = generate("zipf128k", rows=[2])
    s = np.sort(w["p"][0].astype(np.float64))[::-1]
    k = np.arange(1, s.size + 1)
    ratio = s / (k ** -1.1)
    assert np.allclose(ratio, ratio[0], rtol=1e-6)
    assert np.argmax(w["p"][0]) != 0 or np.argmax(generate("zipf128k", rows=[3])["p"][0]) != 0


def test_pair_workload_drafts_follow_their_own_distributions():
    w = generate("pair32k", rows=[0, 1, 2])
    assert w["q2"].shape == w["q"].shape and not np.array_equal(w["q"], w["q2"])
    for i in range(3):
        assert w["q"][i][w["drafts"][i, 0]] > 0 and w["q2"][i][w["drafts"][i, 1]] > 0
    # the second draft is hotter (T = 2.0 vs 1.2): flatter distribution
    ent = lambda a: -(a * np.log(np.maximum(a, 1e-30))).sum(1)
    assert np.all(ent(w["q2"].astype(np.float64)) > ent(w["q"].astype(np.float64)))
