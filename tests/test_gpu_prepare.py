"""sv_prepare_round and the attention's plan / run split, on the GPU.

sv_prepare_round must give exactly what sv_alloc_budget then sv_pack_verify give (bit for
bit: keep, qo_indptr, sel, scores, utilities, tokens, positions, kv_lens; and the budget
and packing oracles' results), and leave in the attention workspace a work plan on which
sv_verify_attn_run reproduces sv_verify_attn bit for bit, run after run: every layer of a
round reuses one plan, so the run must leave it as it found it. sv_verify_attn_plan followed
by runs must do the same.
"""
import numpy as np
import pytest

from gpu_util import say

pytestmark = pytest.mark.gpu

SET_UP = ("keep", "qo", "sel", "scores", "util", "v_tokens", "v_positions", "kv_lens")


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2607_25852_amd import binding
    binding.load()
    return torch


def _snap(torch, rnd, names):
    return {n: getattr(rnd, n).clone() for n in names}


def _poison(rnd, names):
    for n in names:
        t = getattr(rnd, n)
        t.fill_(-3.0 if t.dtype.is_floating_point else -7)


def _same(torch, a, b, what):
    for k in a:
        assert torch.equal(a[k], b[k]), (what, k)


@pytest.mark.parametrize("name", ["tiny", "c16_b16", "c64_b16", "sweep_mtp_c4", "sweep_blk_c32", "sweep_mtp_c64"])
def test_prepare_round_equals_separate_calls(dev, orc, name):
    import torch
    from paper_2607_25852_amd import binding as B, synth
    from paper_2607_25852_amd.round import DeviceRound
    cfg = synth.CONFIGS[name]
    say("prepare", name)
    rnd = DeviceRound(cfg, kind="logits", fused=False, with_accept=False, fill_unused=float("nan"))
    # the separate calls
    rnd.run_budget()
    rnd.run_pack()
    rnd.run_attn()
    torch.cuda.synchronize()
    ref = _snap(torch, rnd, SET_UP + ("attn_out", "attn_lse"))
    # against the oracles: the budget's selection and the packing of its qo_indptr
    conf = rnd.lr["conf"]
    ob = (orc.budget(conf, "fixed", fixed_budget=cfg.budget[1]) if cfg.budget[0] == "fixed"
          else orc.budget(conf, "cost", cost=synth.profiled_cost(cfg.R, cfg.b)))
    np.testing.assert_array_equal(ref["qo"].cpu().numpy(), ob["qo_indptr"])
    tok, pos, kvl = orc.pack_verify(rnd.block_tokens_host, rnd.L, ob["qo_indptr"], cfg.R * cfg.b)
    K = int(ob["qo_indptr"][-1])
    np.testing.assert_array_equal(ref["kv_lens"].cpu().numpy(), kvl)
    np.testing.assert_array_equal(ref["v_tokens"][:K].cpu().numpy(), tok[:K])
    np.testing.assert_array_equal(ref["v_positions"][:K].cpu().numpy(), pos[:K])
    # the fused set-up, then three attention runs on its plan (three layers of one round)
    _poison(rnd, SET_UP + ("attn_out", "attn_lse"))
    rnd.attn_ws.fill_(0xA5)
    rnd.run_prepare()
    for layer in range(3):
        if layer:
            _poison(rnd, ("attn_out", "attn_lse"))
        rnd.run_attn_planned()
        torch.cuda.synchronize()
        got = _snap(torch, rnd, SET_UP + ("attn_out", "attn_lse"))
        # rows past K of the packed batch are not written by either path
        for n in ("v_tokens", "v_positions"):
            got[n], ref_n = got[n][:K], ref[n][:K]
            assert torch.equal(got[n], ref_n), (name, n)
        # utilities: one per candidate ratio (one in fixed mode); the rest of the buffer is not written
        nu = 1 if cfg.budget[0] == "fixed" else len(synth.PAPER_RATIOS_PM)
        got["util"], ref_u = got["util"][:nu], ref["util"][:nu]
        assert torch.equal(got["util"], ref_u), (name, "util")
        skip = ("v_tokens", "v_positions", "attn_out", "attn_lse", "util")
        _same(torch, {k: v for k, v in got.items() if k not in skip}, {k: v for k, v in ref.items() if k not in skip},
              name)
        assert torch.equal(got["attn_out"][:K], ref["attn_out"][:K]), (name, "attn_out", layer)
        assert torch.equal(got["attn_lse"][:K], ref["attn_lse"][:K]), (name, "attn_lse", layer)
    # sv_verify_attn_plan, then runs on that plan
    _poison(rnd, ("attn_out", "attn_lse"))
    rnd.attn_ws.fill_(0x5A)
    B.verify_attn_plan(rnd.adesc, rnd.qo, rnd.kv_lens, rnd.attn_ws)
    for layer in range(2):
        rnd.run_attn_planned()
        torch.cuda.synchronize()
        assert torch.equal(rnd.attn_out[:K], ref["attn_out"][:K]), (name, "plan + run", layer)
        assert torch.equal(rnd.attn_lse[:K], ref["attn_lse"][:K]), (name, "plan + run", layer)


@pytest.mark.parametrize("R,b,total_cut", [(4096, 2, 0), (512, 16, 0), (64, 16, 37), (3, 1, 0), (8, 16, 0),
                                             (65, 1, 0), (43, 3, 5)])
def test_prepare_round_budget_and_packing_edges(dev, orc, R, b, total_cut):
    """The largest budgets (4096 requests; 8192 positions), a packed batch with fewer rows
    than the budget keeps (rows past total_max are dropped and kv_lens keeps L_i), blocks
    of one position, and the edges of the one-wave form (128 positions; 65 positions of one
    token; 129 positions on 512 threads): the fused set-up against the separate calls and
    the oracles."""
    import torch
    from paper_2607_25852_amd import binding as B, synth
    from paper_2607_25852_amd.round import to_dev
    say("prepare edges", R, b, total_cut)
    rng = np.random.default_rng(R * 31 + b)
    conf = rng.random((R, b - 1)).astype(np.float32) ** 0.2
    if b > 1:
        conf[rng.random((R, b - 1)) < 0.05] = 1.0  # ties
    cost = synth.profiled_cost(R, b)
    bdesc = B.budget_desc(R, b, "cost", ratios_pm=synth.PAPER_RATIOS_PM, cost=cost)
    ob = orc.budget(conf, "cost", cost=cost)
    K = int(ob["qo_indptr"][-1])
    total_max = max(1, K - total_cut)
    blk = rng.integers(0, 1 << 20, size=(R, b)).astype(np.int32)
    L = rng.integers(0, 100000, size=R).astype(np.int32)
    pdesc = B.pack_desc(R, b, total_max)
    d_conf, d_blk, d_L = to_dev(conf), to_dev(blk), to_dev(L)

    def outs():
        return dict(keep=torch.full((R,), -7, dtype=torch.int32, device="cuda"),
                    qo=torch.full((R + 1,), -7, dtype=torch.int32, device="cuda"),
                    sel=torch.full((2,), -7, dtype=torch.int32, device="cuda"),
                    scores=torch.full((R * b,), -3.0, dtype=torch.float32, device="cuda"),
                    util=torch.full((B.SV_MAX_RATIOS,), -7, dtype=torch.int64, device="cuda"),
                    tokens=torch.full((total_max,), -7, dtype=torch.int32, device="cuda"),
                    positions=torch.full((total_max,), -7, dtype=torch.int32, device="cuda"),
                    kv_lens=torch.full((R,), -7, dtype=torch.int32, device="cuda"))
    a, f = outs(), outs()
    B.alloc_budget(bdesc, d_conf, a["keep"], a["qo"], a["sel"], a["scores"], a["util"])
    B.pack_verify(pdesc, d_blk, d_L, a["qo"], a["tokens"], a["positions"], a["kv_lens"])
    B.prepare_round(bdesc, d_conf, f["keep"], f["qo"], f["sel"], f["scores"], f["util"], pdesc, d_blk, d_L,
                    f["tokens"], f["positions"], f["kv_lens"])
    torch.cuda.synchronize()
    for k in a:
        if k == "util":
            n = len(synth.PAPER_RATIOS_PM)
            assert torch.equal(a[k][:n], f[k][:n]), k
        else:
            assert torch.equal(a[k], f[k]), k
    np.testing.assert_array_equal(f["qo"].cpu().numpy(), ob["qo_indptr"])
    tok, pos, kvl = orc.pack_verify(blk, L, ob["qo_indptr"], total_max)
    np.testing.assert_array_equal(f["kv_lens"].cpu().numpy(), kvl)
    for got, want in ((f["tokens"].cpu().numpy(), tok), (f["positions"].cpu().numpy(), pos)):
        np.testing.assert_array_equal(got[want >= 0], want[want >= 0])  # the rows written
        assert np.all(got[want < 0] == -7)  # rows no request owns are left alone


def test_attention_run_on_a_workspace_without_its_plan(dev):
    """sv_verify_attn_run on a workspace that holds no plan, or the plan of other inputs:
    the results are unspecified, but the call must succeed and every access stay in bounds.
    The workspace is filled with uniform bytes and with the 8-byte pattern (0x7FFFFFFF, 0),
    which makes the item count the largest int, the work counter 0 and every other work
    item name request 32767 (beyond the last); then the plan of a round with other key
    counts is used. A plan built afterwards must give sv_verify_attn's results bit for bit."""
    import torch
    from paper_2607_25852_amd import binding as B, synth
    from paper_2607_25852_amd.round import DeviceRound
    cfg = synth.CONFIGS["c64_b16"]
    say("attention run without its plan", cfg.name)
    rnd = DeviceRound(cfg, kind="logits", fused=False, with_accept=False)
    rnd.run_attn()
    torch.cuda.synchronize()
    K = rnd.K
    ref_out, ref_lse = rnd.attn_out[:K].clone(), rnd.attn_lse[:K].clone()
    ws32 = rnd.attn_ws.view(torch.int32)
    fills = [("byte", v) for v in (0x00, 0x01, 0x7F, 0xFF)] + [("pattern", None)]
    for kind, v in fills:
        if kind == "byte":
            rnd.attn_ws.fill_(v)
        else:
            ws32[0::2] = 0x7FFFFFFF
            ws32[1::2] = 0
        rnd.run_attn_planned()
        torch.cuda.synchronize()
    # the plan of other inputs: every request's context halved
    qo = rnd.qo.cpu().numpy()
    kv_a = rnd.kv_lens.cpu().numpy()
    k = np.diff(qo)
    kv_b = torch.from_numpy((kv_a - (kv_a - k) // 2).astype(np.int32)).cuda()
    B.verify_attn_plan(rnd.adesc, rnd.qo, kv_b, rnd.attn_ws)
    rnd.run_attn_planned()
    torch.cuda.synchronize()
    # and back: a plan for these inputs restores the exact results
    rnd.attn_out.fill_(-3.0)
    B.verify_attn_plan(rnd.adesc, rnd.qo, rnd.kv_lens, rnd.attn_ws)
    rnd.run_attn_planned()
    torch.cuda.synchronize()
    assert torch.equal(rnd.attn_out[:K], ref_out)
    assert torch.equal(rnd.attn_lse[:K], ref_lse)
