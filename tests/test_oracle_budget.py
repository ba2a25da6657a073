"""Pins of the D-cut budget oracle (Sec. 4.2) against facts the paper and the
mathematics fix, independent of the oracle's own code:

* eq. dcut-score: fp32 prefix products equal the exact products up to fp32
  rounding, start at 1 and never increase (c in [0,1]);
* greedy top-K over prefix scores is optimal for the estimated batch progress
  (eqs. dcut-expected-advance / dcut-batch-utility), checked by brute force over
  every keep-vector on tiny batches;
* the shallow-first tie rule keeps contiguous prefixes; further ties go to the
  lower request index (our reading, the paper only fixes depth);
* eq. dcut-budget: K_rho = max(B, ceil(rho*B*(D+1))); rho = 1 keeps whole blocks;
* eq. dcut-select: argmax U/C, hand-worked examples in tests/golden/.
"""
import itertools
import json
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_conf(rng, R, D, p_one=0.1, p_zero=0.05):
    c = rng.random((R, D)).astype(np.float32)
    c[rng.random((R, D)) < p_one] = 1.0
    c[rng.random((R, D)) < p_zero] = 0.0
    return c


def test_scores_are_prefix_products(orc):
    rng = np.random.default_rng(1)
    conf = _rand_conf(rng, 50, 15)
    s = orc.prefix_scores(conf)
    assert s.shape == (50, 16) and s.dtype == np.float32
    assert np.all(s[:, 0] == 1.0)
    exact = np.concatenate([np.ones((50, 1)), np.cumprod(conf.astype(np.float64), axis=1)], axis=1)
    k = np.arange(16)[None, :]
    # k fp32 roundings, each at most 2^-24 relative
    assert np.all(np.abs(s - exact) <= k * 2.0 ** -24 * exact + 1e-45)
    assert np.all(np.diff(s, axis=1) <= 0.0)


def test_scores_sanitise_out_of_range_confidence(orc):
    conf = np.array([[np.nan, 0.5], [-1.0, 0.5], [2.0, 0.5], [0.5, np.inf]], np.float32)
    s = orc.prefix_scores(conf)
    np.testing.assert_array_equal(s, np.array(
        [[1, 0, 0], [1, 0, 0], [1, 1, 0.5], [1, 0.5, 0.5]], np.float32))


def _fixed(s):
    return int(np.float64(s) * 2.0 ** 40)


@pytest.mark.parametrize("R,D", [(1, 3), (2, 2), (2, 3), (3, 2), (3, 3)])
def test_topk_is_optimal_by_brute_force(orc, R, D):
    """For every K, the oracle's keep-vector attains the maximum of
    sum_i sum_{k<=n_i} s_{i,k} over all keep-vectors with sum(n_i+1) = K."""
    rng = np.random.default_rng(100 + 10 * R + D)
    b = D + 1
    for trial in range(30):
        conf = _rand_conf(rng, R, D, p_one=0.2, p_zero=0.1)
        if trial % 5 == 0:  # many exact ties
            conf = rng.choice(np.array([0.0, 0.25, 0.5, 1.0], np.float32), size=(R, D))
        s = orc.prefix_scores(conf)
        fx = [[_fixed(s[i, k]) for k in range(b)] for i in range(R)]
        for K in range(R, R * b + 1):
            res = orc.budget(conf, mode="fixed", fixed_budget=K)
            keep = res["keep"]
            assert keep.sum() + R == K and np.all(keep >= 0) and np.all(keep <= D)
            got = sum(sum(fx[i][:keep[i] + 1]) for i in range(R))
            assert got == int(res["utility"][0])
            best = 0
            for nv in itertools.product(range(b), repeat=R):
                if sum(nv) + R != K:
                    continue
                best = max(best, sum(sum(fx[i][:nv[i] + 1]) for i in range(R)))
            assert got == best, (conf, K, keep)


def test_tie_breaks_shallow_then_lower_request(orc):
    # all confidences 1: every score is 1; the order is depth first, then request
    conf = np.ones((3, 3), np.float32)
    for K, want in [(3, [0, 0, 0]), (4, [1, 0, 0]), (5, [1, 1, 0]), (6, [1, 1, 1]),
                    (7, [2, 1, 1]), (9, [2, 2, 2]), (12, [3, 3, 3])]:
        np.testing.assert_array_equal(orc.budget(conf, "fixed", K)["keep"], want)
    # equal rows in two requests, a distinct third
    conf = np.array([[0.5, 0.5], [0.5, 0.5], [0.9, 0.9]], np.float32)
    # scores: r0,r1 = 1,.5,.25 ; r2 = 1,.9,.81
    for K, want in [(4, [0, 0, 1]), (5, [0, 0, 2]), (6, [1, 0, 2]), (7, [1, 1, 2]), (8, [2, 1, 2])]:
        np.testing.assert_array_equal(orc.budget(conf, "fixed", K)["keep"], want)


def test_contiguous_prefixes_and_invariants(orc):
    rng = np.random.default_rng(7)
    for trial in range(40):
        R = int(rng.integers(1, 40))
        D = int(rng.integers(1, 16))
        conf = _rand_conf(rng, R, D)
        cost = np.sort(rng.integers(1000, 100000, size=4)).astype(np.uint32)
        res = orc.budget(conf, "cost", cost=cost)
        s = res["scores"]
        keep = res["keep"]
        K = res["K"]
        assert R <= K <= R * (D + 1)
        assert keep.sum() + R == K
        assert res["qo_indptr"][0] == 0 and np.all(np.diff(res["qo_indptr"]) == keep + 1)
        # selected set == top-K by the stated order: every kept score >= every dropped one
        kept = np.concatenate([s[i, :keep[i] + 1] for i in range(R)])
        dropped = np.concatenate([s[i, keep[i] + 1:] for i in range(R)])
        if len(dropped):
            assert kept.min() >= dropped.max()
        # eq. dcut-budget and monotonicity in rho
        Ks = [max(R, -(-pm * R * (D + 1) // 1000)) for pm in (250, 500, 750, 1000)]
        assert K == Ks[res["rho_index"]]
        U = [int(u) for u in res["utility"]]
        assert U == sorted(U)


def test_ratio_one_keeps_everything(orc):
    rng = np.random.default_rng(3)
    conf = _rand_conf(rng, 9, 7)
    res = orc.budget(conf, "cost", ratios_pm=(1000,), cost=[5])
    assert res["K"] == 9 * 8 and np.all(res["keep"] == 7) and res["rho_index"] == 0
    res = orc.budget(conf, "fixed", fixed_budget=72)
    assert np.all(res["keep"] == 7)


def test_lower_bound_keeps_every_certain_token(orc):
    conf = np.zeros((5, 4), np.float32)
    res = orc.budget(conf, "cost", ratios_pm=(100,), cost=[1])  # ceil(0.1*25)=3 < R=5
    assert res["K"] == 5 and np.all(res["keep"] == 0)


@pytest.mark.parametrize("case", json.load(open(os.path.join(GOLDEN, "dcut_select_cases.json")))["cases"],
                         ids=lambda c: c["name"])
def test_select_golden(orc, case):
    conf = np.array(case["conf"], np.float32)
    res = orc.budget(conf, "cost", ratios_pm=case["ratios_pm"], cost=case["cost"])
    assert res["rho_index"] == case["rho_index"]
    assert res["K"] == case["K"]
    np.testing.assert_array_equal(res["keep"], case["keep"])
    np.testing.assert_array_equal(res["qo_indptr"], case["qo_indptr"])
    assert [int(u) for u in res["utility"]] == case["utility_fixed"]


def test_invalid_arguments_are_rejected(orc):
    conf = np.ones((2, 2), np.float32)
    with pytest.raises(ValueError):
        orc.budget(conf, "fixed", fixed_budget=1)  # below R
    with pytest.raises(ValueError):
        orc.budget(conf, "fixed", fixed_budget=7)  # above R*b


def test_full_budget_keeps_everything(orc):
    """FIXED mode with K = R*b (the tiny and c16_b16 workloads) selects every position:
    n_i = D for all requests and qo_indptr = (0, b, 2b, ...)."""
    from paper_2607_25852_amd import synth
    for name in ("tiny", "c16_b16"):
        cfg = synth.CONFIGS[name]
        assert cfg.budget == ("fixed", cfg.R * cfg.b)
        conf = synth.make_logits_round(cfg)["conf"]
        res = orc.budget(conf, "fixed", fixed_budget=cfg.R * cfg.b)
        assert (np.asarray(res["keep"]) == cfg.b - 1).all()
        np.testing.assert_array_equal(res["qo_indptr"], np.arange(cfg.R + 1) * cfg.b)
