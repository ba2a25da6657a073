"""sv_draft_stats and sv_spec_accept_stats on the GPU.

sv_draft_stats against the fp64 oracle: m within fp32 rounding of l/T, S and the
confidence within a relative 2e-5 (S is an fp32 sum of up to 2^22 terms).
sv_spec_accept_stats with statistics from sv_draft_stats against sv_spec_accept on the
same inputs: bit-identical accepted lengths, tokens and flags (both use the same chunk
statistics and merge), at the small workloads and at the full c64_b16 round; and against
the oracle with the logits-mode rule of the acceptance tests.
"""
import numpy as np
import pytest

import oracle
from gpu_util import classify_accept, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2607_25852_amd import binding
    binding.load()
    return torch


def gpu_draft_stats(torch, draft, dtype, T=1.0):
    from paper_2607_25852_amd import binding as B
    from paper_2607_25852_amd.round import to_dev
    R, D, V = draft.shape
    d = B.draft_stats_desc(R, D, V, B.SV_F32 if dtype == "f32" else B.SV_BF16, T)
    ws = torch.empty(max(B.draft_stats_workspace_size(d), 256), dtype=torch.uint8, device="cuda")
    stats = torch.full((R * D, 2), float("nan"), dtype=torch.float32, device="cuda")
    conf = torch.full((R * D,), float("nan"), dtype=torch.float32, device="cuda")
    B.draft_stats(d, to_dev(draft), stats, conf, ws)
    torch.cuda.synchronize()
    return stats, conf


def check_stats(stats, conf, draft, dtype, T):
    ref = oracle.draft_stats(draft, temperature=T, dtype=dtype)
    st = stats.cpu().numpy().astype(np.float64)
    m, S, c = st[:, 0], st[:, 1], conf.cpu().numpy().astype(np.float64)
    np.testing.assert_allclose(m, ref["m"].reshape(-1), rtol=3e-7, atol=0)
    np.testing.assert_allclose(S, ref["S"].reshape(-1), rtol=2e-5)
    np.testing.assert_allclose(c, ref["conf"].reshape(-1), rtol=2e-5)


@pytest.mark.parametrize("R,D,V,dtype,T,seed", [
    (1, 1, 1, "f32", 1.0, 0),
    (4, 7, 1024, "f32", 1.0, 1),
    (3, 5, 1000, "f32", 0.7, 2),       # ragged last chunk
    (16, 15, 32768, "bf16", 1.0, 3),
    (5, 4, 50001, "bf16", 1.3, 4),     # ragged, odd vocabulary
    (2, 3, 1 << 22, "bf16", 1.0, 5),   # the largest vocabulary
])
def test_draft_stats_vs_oracle(dev, R, D, V, dtype, T, seed):
    from paper_2607_25852_amd import synth
    say(f"draft stats R={R} D={D} V={V} {dtype} T={T}")
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal((R, D, V), dtype=np.float32) * np.float32(3.0))
    if R * D > 1:
        x[0, 0, :] = 0.0                 # uniform row: S = V, conf = 1/V
        x[-1, -1, rng.integers(0, V)] = 40.0  # one dominant logit: conf near 1
    draft = x if dtype == "f32" else synth.bf16_bits(x)
    stats, conf = gpu_draft_stats(dev, draft, dtype, T)
    check_stats(stats, conf, draft, dtype, T)


def _round(name):
    from test_gpu_accept import _workload
    return _workload(name, "logits")


def _accept_both(torch, cfg, target, draft, tokens, qo, ua, us, dtype):
    from paper_2607_25852_amd import binding as B
    from paper_2607_25852_amd.round import to_dev
    from test_gpu_accept import gpu_accept
    R, D, V = draft.shape
    plain = gpu_accept(torch, target, draft, tokens, qo, ua, us, "logits", dtype)
    stats, conf = gpu_draft_stats(torch, draft, dtype)
    d = B.accept_desc(R, D + 1, V, B.SV_LOGITS, B.SV_F32 if dtype == "f32" else B.SV_BF16)
    ws = torch.empty(B.accept_workspace_size(d), dtype=torch.uint8, device="cuda")
    acc = torch.full((R,), -9, dtype=torch.int32, device="cuda")
    out = torch.full((R, D + 1), -9, dtype=torch.int32, device="cuda")
    flags = torch.full((R,), -9, dtype=torch.int32, device="cuda")
    B.spec_accept_stats(d, to_dev(target), to_dev(draft), stats, to_dev(np.ascontiguousarray(tokens, np.int32)),
                        to_dev(np.ascontiguousarray(qo, np.int32)), to_dev(np.ascontiguousarray(ua, np.float32)),
                        to_dev(np.ascontiguousarray(us, np.float32)), acc, out, flags, ws)
    torch.cuda.synchronize()
    with_stats = dict(accept_len=acc.cpu().numpy(), out_tokens=out.cpu().numpy(), flags=flags.cpu().numpy())
    return plain, with_stats, stats, conf


@pytest.mark.parametrize("name", ["tiny", "c16_b16", "c64_b16", "sweep_mtp_c64"])
def test_accept_stats_equals_accept(dev, name):
    say("accept with draft stats", name)
    cfg, target, draft, tokens, qo, ua, us, dtype = _round(name)
    plain, with_stats, stats, conf = _accept_both(dev, cfg, target, draft, tokens, qo, ua, us, dtype)
    for k in ("accept_len", "out_tokens", "flags"):
        np.testing.assert_array_equal(with_stats[k], plain[k], err_msg=k)
    # the drafter's confidences agree with the input generator's own
    from paper_2607_25852_amd import synth
    lr_conf = synth.make_logits_round(cfg)["conf"].reshape(-1) if name == "tiny" else None
    if lr_conf is not None:
        np.testing.assert_allclose(conf.cpu().numpy(), lr_conf, rtol=2e-5)


@pytest.mark.parametrize("name", ["tiny", "c16_b16"])
def test_accept_stats_vs_oracle(dev, orc, name):
    say("accept with draft stats vs oracle", name)
    cfg, target, draft, tokens, qo, ua, us, dtype = _round(name)
    _, with_stats, _, _ = _accept_both(dev, cfg, target, draft, tokens, qo, ua, us, dtype)
    ref = orc.accept(target, draft, tokens, qo, ua, us, kind="logits", dtype=dtype, diagnostics=True)
    exact, marginal, failures = classify_accept(with_stats, ref, ua)
    say("accept with draft stats vs oracle", name, "exact", exact, "marginal", marginal)
    assert not failures, failures[:5]
    assert marginal <= max(1, cfg.R // 50)
