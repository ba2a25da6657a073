"""sv_alloc_budget on the GPU against the oracle: keep depths, qo_indptr, the
selection (K, ratio), scores and utilities must match bit for bit."""
import json
import os

import numpy as np
import pytest

from gpu_util import SWEEP, conf_of, say

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2607_25852_amd import binding
    binding.load()
    return torch


def gpu_budget(torch, conf, mode, fixed=0, ratios=(250, 500, 750, 1000), cost=None):
    from paper_2607_25852_amd import binding as B
    R, D = conf.shape
    b = D + 1
    d = B.budget_desc(R, b, mode, fixed_budget=fixed, ratios_pm=ratios,
                      cost=cost if cost is not None else [1] * len(ratios))
    conf_d = torch.from_numpy(np.ascontiguousarray(conf, np.float32)).cuda() if D > 0 else None
    keep = torch.full((R,), -7, dtype=torch.int32, device="cuda")
    qo = torch.full((R + 1,), -7, dtype=torch.int32, device="cuda")
    sel = torch.full((2,), -7, dtype=torch.int32, device="cuda")
    scores = torch.full((R * b,), -1.0, dtype=torch.float32, device="cuda")
    util = torch.zeros(8, dtype=torch.int64, device="cuda")
    B.alloc_budget(d, conf_d, keep, qo, sel, scores, util)
    torch.cuda.synchronize()
    nr = len(ratios) if mode == "cost" else 1
    return dict(keep=keep.cpu().numpy(), qo_indptr=qo.cpu().numpy(), K=int(sel[0]), rho_index=int(sel[1]),
                scores=scores.cpu().numpy().reshape(R, b),
                utility=util.cpu().numpy().view(np.uint64)[:nr])


def assert_same(g, o):
    np.testing.assert_array_equal(g["keep"], o["keep"])
    np.testing.assert_array_equal(g["qo_indptr"], o["qo_indptr"])
    assert g["K"] == o["K"] and g["rho_index"] == o["rho_index"]
    np.testing.assert_array_equal(g["scores"].view(np.uint32), o["scores"].view(np.uint32))
    np.testing.assert_array_equal(g["utility"], o["utility"])


@pytest.mark.parametrize("name", ["tiny", "c16_b16", "c64_b16"] + SWEEP)
def test_workload_budgets(dev, orc, name):
    from paper_2607_25852_amd import synth
    cfg = synth.CONFIGS[name]
    say("budget workload", name)
    conf = conf_of(name)
    if cfg.budget[0] == "fixed":
        g = gpu_budget(dev, conf, "fixed", fixed=cfg.budget[1])
        o = orc.budget(conf, "fixed", fixed_budget=cfg.budget[1])
    else:
        cost = synth.profiled_cost(cfg.R, cfg.b)
        g = gpu_budget(dev, conf, "cost", cost=cost)
        o = orc.budget(conf, "cost", cost=cost)
    assert_same(g, o)


@pytest.mark.parametrize("case", json.load(open(os.path.join(GOLDEN, "dcut_select_cases.json")))["cases"],
                         ids=lambda c: c["name"])
def test_golden_selection(dev, case):
    say("budget golden", case["name"])
    g = gpu_budget(dev, np.array(case["conf"], np.float32), "cost", ratios=case["ratios_pm"], cost=case["cost"])
    assert g["rho_index"] == case["rho_index"] and g["K"] == case["K"]
    np.testing.assert_array_equal(g["keep"], case["keep"])
    np.testing.assert_array_equal(g["qo_indptr"], case["qo_indptr"])
    assert [int(u) for u in g["utility"]] == case["utility_fixed"]


def _conf(rng, R, D, style):
    if style == "ties":
        return rng.choice(np.array([0.0, 0.25, 0.5, 1.0], np.float32), size=(R, D))
    c = rng.random((R, D)).astype(np.float32)
    if style == "dirty":
        m = rng.random((R, D))
        c[m < 0.05] = np.nan
        c[(m >= 0.05) & (m < 0.1)] = -0.5
        c[(m >= 0.1) & (m < 0.15)] = 3.0
        c[(m >= 0.15) & (m < 0.3)] = 1.0
    return c


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("style", ["plain", "ties", "dirty"])
def test_random_budgets(dev, orc, seed, style):
    rng = np.random.default_rng(1000 + seed)
    R = int(rng.integers(1, 300))
    D = int(rng.integers(0, 16))
    conf = _conf(rng, R, D, style)
    say("budget random", style, seed, R, D)
    for mode in ("fixed", "cost"):
        if mode == "fixed":
            K = int(rng.integers(R, R * (D + 1) + 1))
            g, o = gpu_budget(dev, conf, "fixed", fixed=K), orc.budget(conf, "fixed", fixed_budget=K)
        else:
            nr = int(rng.integers(1, 9))
            ratios = tuple(sorted(rng.choice(np.arange(1, 1001), size=nr, replace=False).tolist()))
            cost = rng.integers(1, 1 << 32, size=nr, dtype=np.uint64).astype(np.uint32)
            g = gpu_budget(dev, conf, "cost", ratios=ratios, cost=cost)
            o = orc.budget(conf, "cost", ratios_pm=ratios, cost=cost)
        assert_same(g, o)


@pytest.mark.parametrize("R,D", [(64, 0), (13, 4), (8, 15), (16, 7), (43, 2), (128, 0), (129, 0)])
@pytest.mark.parametrize("style", ["ties", "dirty"])
def test_one_wave_boundaries(dev, orc, R, D, style):
    """Rounds at the edges of the one-wave form of the budget kernel (R*b of 64 and 65, of
    128, and 129, the first that runs on 512 threads) with tied and dirty confidences: every
    budget equals the oracle's bit for bit, in both modes."""
    rng = np.random.default_rng(R * 97 + D)
    conf = _conf(rng, R, D, style)
    say("budget one-wave edge", R, D, style)
    cost = np.array([20000, 21000, 23000, 26000], np.uint32)
    assert_same(gpu_budget(dev, conf, "cost", cost=cost), orc.budget(conf, "cost", cost=cost))
    for K in (R, (R * (D + 1) + R) // 2, R * (D + 1)):
        assert_same(gpu_budget(dev, conf, "fixed", fixed=K), orc.budget(conf, "fixed", fixed_budget=K))


@pytest.mark.parametrize("R,D", [(1, 0), (1, 15), (512, 15), (4096, 1), (2730, 2), (64, 15)])
def test_size_limits(dev, orc, R, D):
    rng = np.random.default_rng(R * 31 + D)
    conf = _conf(rng, R, D, "ties" if R > 1000 else "plain")
    say("budget size", R, D)
    cost = np.array([20000, 21000, 23000, 26000], np.uint32)
    assert_same(gpu_budget(dev, conf, "cost", cost=cost), orc.budget(conf, "cost", cost=cost))
    K = R * (D + 1)
    assert_same(gpu_budget(dev, conf, "fixed", fixed=K), orc.budget(conf, "fixed", fixed_budget=K))
    assert_same(gpu_budget(dev, conf, "fixed", fixed=R), orc.budget(conf, "fixed", fixed_budget=R))


def test_repeatable(dev):
    rng = np.random.default_rng(5)
    conf = _conf(rng, 200, 15, "ties")
    a = gpu_budget(dev, conf, "cost", cost=[3, 4, 5, 6])
    b = gpu_budget(dev, conf, "cost", cost=[3, 4, 5, 6])
    assert_same(a, b)
