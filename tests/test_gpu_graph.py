"""One HIP graph per round shape.

The whole round -- budget, packing of the verify batch (key counts), attention and
acceptance -- is captured once and replayed. Launch shapes depend only on the
descriptors (R, b, vocabulary, heads), never on the budget's choice, which stays on the
device: so one graph serves every choice of that shape. Every replay, with eager work
and synchronisations between replays, must equal the eager round bit for bit and match
the oracle (budget and packing bit-exact, attention within the bf16 tolerance on every
head of the first and last kept row of every request, acceptance under the logits-mode
contract); the same graph must follow new confidences (the requests' confidence rows
permuted: the same utilities and K, a different allocation across requests); and one
graph holding several rounds back to back (one per input copy) must give each copy the
eager result.
"""
import numpy as np
import pytest

from gpu_util import bf16_bits_of, classify_accept, compare_attention, f32_of_bits, say

pytestmark = pytest.mark.gpu

OUTS = ("sel", "qo", "keep", "kv_lens", "v_tokens", "v_positions", "attn_out", "attn_lse", "accept_len",
        "out_tokens", "flags")


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2607_25852_amd import binding
    binding.load()
    return torch


def poison(rnd):
    for name in OUTS:
        t = getattr(rnd, name)
        if t.dtype.is_floating_point:
            t.fill_(-3.0)
        else:
            t.fill_(-7)


def snapshot(rnd):
    return {name: getattr(rnd, name).clone() for name in OUTS}


def same(x, y):
    import torch
    for k in x:
        assert torch.equal(x[k], y[k]), k


def check_with_oracle(rnd, snap, conf):
    """The outputs of one round (a graph replay's snapshot) against the oracle."""
    import oracle
    from paper_2607_25852_amd import synth
    cfg = rnd.cfg
    ob = oracle.budget(conf, "cost", cost=synth.profiled_cost(cfg.R, cfg.b))
    qo = ob["qo_indptr"]
    K = int(qo[-1])
    np.testing.assert_array_equal(snap["qo"].cpu().numpy(), qo)
    np.testing.assert_array_equal(snap["keep"].cpu().numpy(), ob["keep"])
    assert int(snap["sel"][0]) == K
    o_tok, o_pos, o_kvl = oracle.pack_verify(rnd.block_tokens_host, rnd.L, qo, cfg.R * cfg.b)
    np.testing.assert_array_equal(snap["kv_lens"].cpu().numpy(), o_kvl)
    np.testing.assert_array_equal(snap["v_tokens"][:K].cpu().numpy(), o_tok[:K])
    np.testing.assert_array_equal(snap["v_positions"][:K].cpu().numpy(), o_pos[:K])
    # attention: every head of the first and last kept row of every request. The query rows
    # the round holds were packed for the first selection; the oracle reads the same rows.
    q_rows = bf16_bits_of(rnd.q)
    first, last = qo[:-1], qo[1:] - 1
    rows = np.unique(np.concatenate([first, last])).astype(np.int32)
    units = (np.repeat(rows, cfg.Hq).astype(np.int32), np.tile(np.arange(cfg.Hq, dtype=np.int32), len(rows)))
    o_ref, l_ref = oracle.attention(q_rows[:K], rnd.kv["k_cache"], rnd.kv["v_cache"], rnd.kv["page_table"], qo,
                                    o_kvl, dtype="bf16", units=units)
    out = f32_of_bits(bf16_bits_of(snap["attn_out"]))
    lse = snap["attn_lse"].cpu().numpy()
    ok, info = compare_attention(out[units[0], units[1]], lse[units[0], units[1]], o_ref, l_ref, "bf16")
    say("graph replay attention vs oracle", info)
    assert ok, info
    # acceptance on the target rows the round holds (packed for the first selection)
    oa = oracle.accept(rnd.target_host, rnd.draft_host, rnd.lr["draft_tokens"], qo, rnd.ua_host, rnd.us_host,
                       kind="logits", dtype="bf16", diagnostics=True)
    g = dict(accept_len=snap["accept_len"].cpu().numpy(), out_tokens=snap["out_tokens"].cpu().numpy())
    exact, marginal, failures = classify_accept(g, oa, rnd.ua_host)
    say("graph replay acceptance vs oracle: exact", exact, "marginal", marginal)
    assert not failures, failures[:5]
    assert marginal <= max(1, cfg.R // 50)


def test_round_graph_replays_and_follows_the_budget(dev):
    torch = dev
    from paper_2607_25852_amd import synth
    from paper_2607_25852_amd.round import DeviceRound, to_dev
    cfg = synth.CONFIGS["c64_b16"]
    say("graph round", cfg.name)
    rnd = DeviceRound(cfg, kind="logits")
    R = cfg.R

    poison(rnd)
    rnd.run()
    torch.cuda.synchronize()
    ref = snapshot(rnd)
    # capture (warm-up on the capture stream first)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        rnd.run()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        rnd.run()
    torch.cuda.synchronize()
    for rep in range(3):
        poison(rnd)
        x = torch.randn(1 << 20, device="cuda")
        float((x * x).sum())  # eager work and a synchronisation between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        snap = snapshot(rnd)
        same(snap, ref)
        if rep == 0:
            check_with_oracle(rnd, snap, rnd.lr["conf"])
    # new confidences: permute the requests' rows (same utilities and K, other allocation)
    perm = np.random.default_rng(3).permutation(R)
    conf2 = np.ascontiguousarray(rnd.lr["conf"][perm])
    rnd.conf.copy_(to_dev(conf2))
    poison(rnd)
    rnd.run()
    torch.cuda.synchronize()
    ref2 = snapshot(rnd)
    assert torch.equal(ref2["sel"], ref["sel"]) and int(ref2["qo"][-1]) == int(ref["qo"][-1])
    assert not torch.equal(ref2["qo"], ref["qo"])
    for rep in range(2):
        poison(rnd)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        snap = snapshot(rnd)
        same(snap, ref2)
        if rep == 0:
            check_with_oracle(rnd, snap, conf2)


def test_several_rounds_in_one_graph(dev):
    """Rounds on three input copies captured back to back in one graph: each copy gets the
    eager round's outputs on every replay."""
    torch = dev
    from paper_2607_25852_amd import synth
    from paper_2607_25852_amd.round import DeviceRound
    cfg = synth.CONFIGS["sweep_blk_c16"]
    say("graph chain", cfg.name)
    base = DeviceRound(cfg, kind="logits", kv="device")
    rounds = [base, base.replica(), base.replica()]
    for r in rounds:
        poison(r)
        r.run()
    torch.cuda.synchronize()
    refs = [snapshot(r) for r in rounds]
    for r in rounds[1:]:
        same(snapshot(r), refs[0])
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for r in rounds:
            r.run()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for r in rounds:
            r.run()
    torch.cuda.synchronize()
    for rep in range(3):
        for r in rounds:
            poison(r)
        x = torch.randn(1 << 20, device="cuda")
        float((x * x).sum())
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for r, ref in zip(rounds, refs):
            same(snapshot(r), ref)
