"""One HIP graph per round shape.

The whole round -- budget, packing of the verify batch (key counts), attention and
acceptance -- is captured once and replayed. Launch shapes depend only on the
descriptors (R, b, vocabulary, heads), never on the budget's choice, which stays on the
device: so one graph serves every choice of that shape. Every replay, with eager work
and synchronisations between replays, must equal the eager round bit for bit; and the
same graph must follow new confidences (the requests' confidence rows permuted: the same
utilities and K, a different allocation across requests).
"""
import numpy as np
import pytest

from gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2607_25852_amd import binding
    binding.load()
    return torch


def test_round_graph_replays_and_follows_the_budget(dev):
    torch = dev
    from paper_2607_25852_amd import binding as B
    from paper_2607_25852_amd import synth
    from paper_2607_25852_amd.round import DeviceRound, to_dev
    cfg = synth.CONFIGS["c64_b16"]
    say("graph round", cfg.name)
    rnd = DeviceRound(cfg, kind="logits")
    R, b = cfg.R, cfg.b
    ctx = to_dev(np.asarray(rnd.L, np.int32))
    blk = to_dev(np.arange(R * b, dtype=np.int32).reshape(R, b))
    p_tok = torch.empty(R * b, dtype=torch.int32, device="cuda")
    p_pos = torch.empty(R * b, dtype=torch.int32, device="cuda")
    pdesc = B.pack_desc(R, b, R * b)

    def round_():
        rnd.run_budget()
        B.pack_verify(pdesc, blk, ctx, rnd.qo, p_tok, p_pos, rnd.kv_lens)  # kv_lens = L + k from the budget
        rnd.run_attn()
        rnd.run_accept()

    outs = ("sel", "qo", "keep", "kv_lens", "attn_out", "attn_lse", "accept_len", "out_tokens", "flags")

    def poison():
        for name in outs:
            t = getattr(rnd, name)
            if t.dtype.is_floating_point:
                t.fill_(-3.0)
            else:
                t.fill_(-7)
        p_pos.fill_(-7)

    def snapshot():
        d = {name: getattr(rnd, name).clone() for name in outs}
        d["p_pos"] = p_pos.clone()
        return d

    def same(x, y):
        for k in x:
            assert torch.equal(x[k], y[k]), k

    poison()
    round_()
    torch.cuda.synchronize()
    ref = snapshot()
    # capture (warm-up on the capture stream first)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        round_()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        round_()
    torch.cuda.synchronize()
    for rep in range(3):
        poison()
        x = torch.randn(1 << 20, device="cuda")
        float((x * x).sum())  # eager work and a synchronisation between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        same(snapshot(), ref)
    # new confidences: permute the requests' rows (same utilities and K, other allocation)
    perm = np.random.default_rng(3).permutation(R)
    rnd.conf.copy_(to_dev(np.ascontiguousarray(rnd.lr["conf"][perm])))
    poison()
    round_()
    torch.cuda.synchronize()
    ref2 = snapshot()
    assert torch.equal(ref2["sel"], ref["sel"]) and int(ref2["qo"][-1]) == int(ref["qo"][-1])
    assert not torch.equal(ref2["qo"], ref["qo"])
    for rep in range(2):
        poison()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        same(snapshot(), ref2)
