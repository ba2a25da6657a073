"""Whole rounds on randomly drawn shapes, through the calls a serving engine makes per
round: sv_prepare_round (budget, packing, attention plan), sv_verify_attn_run and
sv_spec_accept, with every output checked against the oracles:
- the budget's keep/qo_indptr/selection and the packed batch bit for bit;
- attention on sampled (row, head) units that cover every request, both ends of every
  block and every head, at the bf16 / fp32 gates;
- acceptance under the logits-mode contract margins.
The shapes vary what the named workloads hold fixed: GQA group 1-16 (whole-tile waves
above 128 rows per kv-head group), head dim 64/128, pages of 1-128 tokens, contexts from
0 to 2000 keys, vocabularies of 2-6000, bf16 and fp32, cost-table and fixed budgets,
and the temperature of acceptance (1, 0 = greedy verification, 0.6, 1.7).
Unowned pages and slots hold NaN. Seeded; each case names its shape before its GPU step.
"""
import numpy as np
import pytest

from gpu_util import classify_accept, compare_attention, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2607_25852_amd import binding
    binding.load()
    return torch


def _draw(seed):
    from paper_2607_25852_amd import synth
    rng = np.random.default_rng(5000 + seed)
    R = int(rng.integers(1, 33))
    b = int(rng.integers(2, 17))
    Hkv = int(rng.choice([1, 2, 4, 8]))
    G = int(rng.choice([g for g in (1, 2, 4, 8, 16) if g * Hkv <= 64]))
    d = int(rng.choice([64, 128]))
    page = int(rng.choice([1, 16, 32, 64, 128]))
    V = int(rng.integers(2, 6001))
    if seed % 5 == 2:  # more than 128 rows per kv-head group: whole-tile waves
        G, Hkv, b = 16, int(rng.choice([1, 2, 4])), int(rng.integers(9, 17))
    lo = 0 if seed % 7 == 3 else int(rng.integers(0, 1500))
    hi = lo + int(rng.integers(0, 500))
    dtype = "f32" if seed % 4 == 0 else "bf16"
    budget = ("fixed", int(rng.integers(R, R * b + 1))) if seed % 3 == 0 else ("cost",)
    logits = ("plain", float(rng.uniform(0.5, 4.0)), float(rng.uniform(0.1, 2.0)))
    return synth.RoundConfig(f"random{seed}", R, b, V, dtype, G * Hkv, Hkv, d, page, ("uniform", lo, hi), logits,
                             budget, 9000 + seed)


TEMPERATURES = (1.0, 0.0, 0.6, 1.0, 1.7, 1.0)


@pytest.mark.parametrize("seed", range(48))
def test_random_round(dev, orc, seed):
    import torch
    from paper_2607_25852_amd import binding as B, synth
    from paper_2607_25852_amd.round import DeviceRound
    cfg = _draw(seed)
    T = TEMPERATURES[seed % len(TEMPERATURES)]
    say("random round", seed, cfg, "T", T)
    rnd = DeviceRound(cfg, kind="logits", fill_unused=float("nan"))
    if T != 1.0:
        rnd.xdesc = B.accept_desc(cfg.R, cfg.b, cfg.V, B.SV_LOGITS, B.SV_F32 if cfg.dtype == "f32" else B.SV_BF16,
                                  temperature=T)
        rnd.acc_ws = torch.empty(max(B.accept_workspace_size(rnd.xdesc), 256), dtype=torch.uint8, device="cuda")
    for name in ("keep", "qo", "kv_lens", "attn_out", "attn_lse", "accept_len", "out_tokens"):
        t = getattr(rnd, name)
        t.fill_(float("nan") if t.dtype.is_floating_point else -7)
    rnd.run()
    torch.cuda.synchronize()
    R, b = cfg.R, cfg.b
    # budget and packing: bit for bit
    conf = rnd.lr["conf"]
    ob = (orc.budget(conf, "fixed", fixed_budget=cfg.budget[1]) if cfg.budget[0] == "fixed"
          else orc.budget(conf, "cost", cost=synth.profiled_cost(R, b)))
    qo = ob["qo_indptr"]
    np.testing.assert_array_equal(rnd.qo.cpu().numpy(), qo)
    np.testing.assert_array_equal(rnd.keep.cpu().numpy(), ob["keep"])
    tok, pos, kvl = orc.pack_verify(rnd.block_tokens_host, rnd.L, qo, R * b)
    K = int(qo[-1])
    np.testing.assert_array_equal(rnd.kv_lens.cpu().numpy(), kvl)
    np.testing.assert_array_equal(rnd.v_tokens[:K].cpu().numpy(), tok[:K])
    np.testing.assert_array_equal(rnd.v_positions[:K].cpu().numpy(), pos[:K])
    # attention: rows at both ends of every block and a few inside, every head of each
    rng = np.random.default_rng(seed)
    rows = []
    for i in range(R):
        r0, r1 = int(qo[i]), int(qo[i + 1])
        rows += sorted({r0, r1 - 1, *rng.integers(r0, r1, size=2).tolist()})
    rows = np.repeat(np.array(rows, np.int32), cfg.Hq)
    heads = np.tile(np.arange(cfg.Hq, dtype=np.int32), len(rows) // cfg.Hq)
    qk = synth.pack_rows(rnd.kv["q_full"], qo)
    ref_o, ref_l = orc.attention(qk, rnd.kv["k_cache"], rnd.kv["v_cache"], rnd.kv["page_table"], qo, kvl,
                                 dtype=cfg.dtype, units=(rows, heads))
    out = rnd.attn_out.float().cpu().numpy().astype(np.float64)
    lse = rnd.attn_lse.cpu().numpy().astype(np.float64)
    ok, stats = compare_attention(out[rows, heads], lse[rows, heads], ref_o, ref_l, cfg.dtype)
    say("random round", seed, "attention", stats)
    assert ok, stats
    # acceptance: greedy verification bit for bit (argmax, no arithmetic); sampling under the
    # contract margins (probability rows of the logits, then the draw)
    o = orc.accept(rnd.target_host, rnd.draft_host, rnd.lr["draft_tokens"], qo, rnd.ua_host, rnd.us_host,
                   kind="logits", dtype=cfg.dtype, temperature=T, diagnostics=T != 0.0)
    g = dict(accept_len=rnd.accept_len.cpu().numpy(), out_tokens=rnd.out_tokens.cpu().numpy(),
             flags=rnd.flags.cpu().numpy())
    if T == 0.0:
        np.testing.assert_array_equal(g["accept_len"], o["accept_len"])
        np.testing.assert_array_equal(g["out_tokens"], o["out_tokens"])
        np.testing.assert_array_equal(g["flags"], o["flags"])
        return
    exact, marginal, failures = classify_accept(g, o, rnd.ua_host)
    say("random round", seed, "acceptance exact", exact, "marginal", marginal)
    assert not failures, failures[:5]
    assert marginal <= 1
    assert np.all(g["accept_len"] <= np.diff(qo) - 1)


@pytest.mark.parametrize("seed", range(100, 116))
def test_random_round_probability_rows(dev, orc, seed):
    """The same random rounds with fp32 probability rows: acceptance must equal the
    oracle bit for bit (no rounding separates the two sides)."""
    import torch
    from paper_2607_25852_amd import synth
    from paper_2607_25852_amd.round import DeviceRound
    cfg = _draw(seed)
    say("random round, probability rows", seed, cfg)
    rnd = DeviceRound(cfg, kind="probs", fill_unused=float("nan"))
    rnd.accept_len.fill_(-7)
    rnd.out_tokens.fill_(-7)
    rnd.run()
    torch.cuda.synchronize()
    conf = rnd.lr["conf"]
    ob = (orc.budget(conf, "fixed", fixed_budget=cfg.budget[1]) if cfg.budget[0] == "fixed"
          else orc.budget(conf, "cost", cost=synth.profiled_cost(cfg.R, cfg.b)))
    qo = ob["qo_indptr"]
    np.testing.assert_array_equal(rnd.qo.cpu().numpy(), qo)
    o = orc.accept(rnd.target_host, rnd.draft_host, rnd.lr["draft_tokens"], qo, rnd.ua_host, rnd.us_host,
                   kind="probs")
    np.testing.assert_array_equal(rnd.accept_len.cpu().numpy(), o["accept_len"])
    np.testing.assert_array_equal(rnd.out_tokens.cpu().numpy(), o["out_tokens"])
    np.testing.assert_array_equal(rnd.flags.cpu().numpy(), o["flags"])


@pytest.mark.parametrize("seed", range(200, 216))
def test_random_round_with_draft_statistics(dev, seed):
    """The drafter's side of the random rounds: sv_draft_stats on the draft rows against
    the oracle (m, S and the confidence), then sv_spec_accept_stats with those statistics
    equal to sv_spec_accept on the same inputs, bit for bit, at T = 1, 0.6 and 1.7."""
    import torch
    from paper_2607_25852_amd import binding as B
    from paper_2607_25852_amd.round import DeviceRound
    from test_gpu_draft_stats import check_stats
    cfg = _draw(seed)
    T = (1.0, 0.6, 1.7, 1.0)[seed % 4]
    say("random round, draft statistics", seed, cfg, "T", T)
    rnd = DeviceRound(cfg, kind="logits", with_attn=False)
    R, b, V = cfg.R, cfg.b, cfg.V
    D = b - 1
    dt = B.SV_F32 if cfg.dtype == "f32" else B.SV_BF16
    dsd = B.draft_stats_desc(R, D, V, dt, T)
    dws = torch.empty(max(B.draft_stats_workspace_size(dsd), 256), dtype=torch.uint8, device="cuda")
    stats = torch.full((R * D, 2), float("nan"), dtype=torch.float32, device="cuda")
    conf = torch.full((R * D,), float("nan"), dtype=torch.float32, device="cuda")
    B.draft_stats(dsd, rnd.draft, stats, conf, dws)
    xd = B.accept_desc(R, b, V, B.SV_LOGITS, dt, temperature=T)
    aws = torch.empty(max(B.accept_workspace_size(xd), 256), dtype=torch.uint8, device="cuda")

    def outs():
        return (torch.full((R,), -9, dtype=torch.int32, device="cuda"),
                torch.full((R, b), -9, dtype=torch.int32, device="cuda"),
                torch.full((R,), -9, dtype=torch.int32, device="cuda"))
    a1, o1, f1 = outs()
    a2, o2, f2 = outs()
    B.spec_accept(xd, rnd.target, rnd.draft, rnd.tokens, rnd.qo, rnd.u_accept, rnd.u_sample, a1, o1, f1, aws)
    B.spec_accept_stats(xd, rnd.target, rnd.draft, stats, rnd.tokens, rnd.qo, rnd.u_accept, rnd.u_sample, a2, o2,
                        f2, aws)
    torch.cuda.synchronize()
    check_stats(stats, conf, rnd.draft_host, cfg.dtype, T)
    for x, y in ((a1, a2), (o1, o2), (f1, f2)):
        assert torch.equal(x, y)
