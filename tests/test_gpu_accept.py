"""sv_spec_accept on the GPU against the oracle.

Probability mode: identical fp32 probability rows and uniforms on both sides, so
accepted lengths, committed tokens and flags must match bit for bit.
Logits mode: the GPU computes softmax in fp32; outputs must match except where
the oracle's own decision sits within 1e-5*p of its boundary or the draw within
2^-20*Z of a CDF step (the parity contract's margins; such decisions are counted,
printed and required to be rare).
Every workload runs with the draft rows of pruned positions and target rows past
the packed batch filled with NaN: the kernels must never read them.
"""
import numpy as np
import pytest

from gpu_util import SWEEP, budget_packing, classify_accept, logits_round, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2607_25852_amd import binding
    binding.load()
    return torch


def poisoned(target, draft, qo, extra_rows=3):
    """Copies in which every row the call must not read holds NaN: the draft rows of
    pruned positions (t >= n_i) and `extra_rows` target rows past the packed batch."""
    nan = np.float32(np.nan) if target.dtype == np.float32 else np.uint16(0x7FC0)
    t = np.concatenate([target, np.full((extra_rows, target.shape[1]), nan, target.dtype)])
    d = draft.copy()
    n = np.diff(qo) - 1
    for i in range(d.shape[0]):
        d[i, n[i]:] = nan
    return t, d


def gpu_accept(torch, target, draft, tokens, qo, ua, us, kind, dtype, T=1.0, repeat=1):
    """target/draft: numpy fp32 or uint16 (bf16 bits)."""
    from paper_2607_25852_amd import binding as B
    from paper_2607_25852_amd.round import to_dev
    R, D, V = draft.shape
    b = D + 1
    d = B.accept_desc(R, b, V, B.SV_PROBS if kind == "probs" else B.SV_LOGITS,
                      B.SV_F32 if dtype == "f32" else B.SV_BF16, T)
    ws = torch.empty(B.accept_workspace_size(d), dtype=torch.uint8, device="cuda")
    tg, dr = to_dev(target), to_dev(draft)
    tk, qd = to_dev(np.ascontiguousarray(tokens, np.int32)), to_dev(np.ascontiguousarray(qo, np.int32))
    uad, usd = to_dev(np.ascontiguousarray(ua, np.float32)), to_dev(np.ascontiguousarray(us, np.float32))
    outs = []
    for _ in range(repeat):
        acc = torch.full((R,), -9, dtype=torch.int32, device="cuda")
        out = torch.full((R, b), -9, dtype=torch.int32, device="cuda")
        flags = torch.full((R,), -9, dtype=torch.int32, device="cuda")
        B.spec_accept(d, tg, dr, tk, qd, uad, usd, acc, out, flags, ws)
        torch.cuda.synchronize()
        outs.append(dict(accept_len=acc.cpu().numpy(), out_tokens=out.cpu().numpy(), flags=flags.cpu().numpy()))
    return outs if repeat > 1 else outs[0]


def assert_exact(g, o):
    np.testing.assert_array_equal(g["accept_len"], o["accept_len"])
    np.testing.assert_array_equal(g["out_tokens"], o["out_tokens"])
    np.testing.assert_array_equal(g["flags"], o["flags"])


def _workload(name, kind):
    from paper_2607_25852_amd import synth
    cfg = synth.CONFIGS[name]
    lr = logits_round(name, kind == "probs")
    qo = budget_packing(name)
    ua, us = synth.acceptance_uniforms(cfg)
    if kind == "probs":
        target = synth.pack_rows(lr["target_probs_full"], qo)
        draft = lr["draft_probs"]
        dtype = "f32"
    else:
        target = synth.pack_rows(lr["target_full"], qo)
        draft = lr["draft"]
        dtype = cfg.dtype
    return cfg, target, draft, lr["draft_tokens"], qo, ua, us, dtype


@pytest.mark.parametrize("name", ["tiny", "c16_b16", "c64_b16", "long_c32"] + SWEEP)
def test_probs_mode_bit_exact(dev, orc, name):
    say("accept probs", name)
    cfg, target, draft, toks, qo, ua, us, dtype = _workload(name, "probs")
    g = gpu_accept(dev, *poisoned(target, draft, qo), toks, qo, ua, us, "probs", "f32")
    o = orc.accept(target, draft, toks, qo, ua, us, kind="probs")
    assert_exact(g, o)
    assert np.all(g["accept_len"] <= np.diff(qo) - 1)


@pytest.mark.parametrize("name", ["tiny", "c16_b16", "c64_b16", "long_c32"] + SWEEP)
def test_logits_mode_matches_oracle(dev, orc, name):
    say("accept logits", name)
    cfg, target, draft, toks, qo, ua, us, dtype = _workload(name, "logits")
    g = gpu_accept(dev, *poisoned(target, draft, qo), toks, qo, ua, us, "logits", dtype)
    o = orc.accept(target, draft, toks, qo, ua, us, kind="logits", dtype=dtype, diagnostics=True)
    exact, marginal, failures = classify_accept(g, o, ua)
    say("accept logits", name, "exact", exact, "marginal", marginal, "fail", len(failures))
    assert not failures, failures[:5]
    assert marginal <= max(1, cfg.R // 50)
    np.testing.assert_array_equal(g["flags"] & 4, o["flags"] & 4)


def _rand_rows(rng, n, V, peaky=False):
    x = rng.gamma(0.3 if peaky else 1.0, size=(n, V)) + 1e-6
    return (x / x.sum(axis=-1, keepdims=True)).astype(np.float32)


@pytest.mark.parametrize("V", [1, 2, 7, 1000, 1023, 8192, 8193, 40000])
@pytest.mark.parametrize("b", [1, 2, 9, 16])
def test_ragged_shapes_probs(dev, orc, V, b):
    rng = np.random.default_rng(V * 17 + b)
    R = 23
    D = b - 1
    k = rng.integers(1, b + 1, size=R)
    qo = np.concatenate([[0], np.cumsum(k)]).astype(np.int32)
    target = _rand_rows(rng, int(qo[-1]), V, peaky=True)
    draft = _rand_rows(rng, R * max(D, 1), V, peaky=True).reshape(R, max(D, 1), V)[:, :D]
    draft = np.ascontiguousarray(draft)
    if D > 0:
        toks = np.stack([[rng.choice(V, p=draft[i, t].astype(np.float64) / draft[i, t].astype(np.float64).sum())
                          for t in range(D)] for i in range(R)]).astype(np.int32)
    else:
        toks = np.zeros((R, 0), np.int32)
    ua = (rng.integers(0, 1 << 24, size=(R, D)) * 2.0 ** -24).astype(np.float32)
    us = (rng.integers(0, 1 << 24, size=R) * 2.0 ** -24).astype(np.float32)
    say("accept ragged", V, b)
    g = gpu_accept(dev, target, draft, toks, qo, ua, us, "probs", "f32")
    o = orc.accept(target, draft, toks, qo, ua, us, kind="probs")
    assert_exact(g, o)


@pytest.mark.parametrize("dtype,V,T", [("f32", 1000, 1.0), ("bf16", 4099, 1.0), ("bf16", 32768, 0.6),
                                       ("f32", 8192, 1.7)])
def test_ragged_logits(dev, orc, dtype, V, T):
    from paper_2607_25852_amd import synth
    rng = np.random.default_rng(V + int(T * 10))
    R, b = 37, 12
    D = b - 1
    k = rng.integers(1, b + 1, size=R)
    qo = np.concatenate([[0], np.cumsum(k)]).astype(np.int32)
    tl = (rng.standard_normal((int(qo[-1]), V)) * 3).astype(np.float32)
    dl = (rng.standard_normal((R, D, V)) * 3).astype(np.float32)
    for i in range(R):  # drafts close to their target rows
        n = k[i] - 1
        dl[i, :n] = tl[qo[i]:qo[i] + n] + rng.standard_normal((n, V)).astype(np.float32) * 0.5
    if dtype == "bf16":
        tl, dl = synth.bf16_bits(tl), synth.bf16_bits(dl)
    toks = rng.integers(0, V, size=(R, D)).astype(np.int32)
    ua = (rng.integers(0, 1 << 24, size=(R, D)) * 2.0 ** -24).astype(np.float32)
    us = (rng.integers(0, 1 << 24, size=R) * 2.0 ** -24).astype(np.float32)
    say("accept ragged logits", dtype, V, T)
    g = gpu_accept(dev, tl, dl, toks, qo, ua, us, "logits", dtype, T)
    o = orc.accept(tl, dl, toks, qo, ua, us, kind="logits", dtype=dtype, temperature=T, diagnostics=True)
    exact, marginal, failures = classify_accept(g, o, ua)
    assert not failures, failures[:5]
    assert marginal <= 1


def test_degenerate_rows(dev, orc):
    """empty residual (fallback to p), all-zero row (no token), out-of-range and
    NaN draft tokens, u = 0, one-hot rows, no drafts kept."""
    V, b = 6, 4
    D = b - 1
    P = np.zeros((8, 4, V), np.float32)
    Q = np.zeros((8, D, V), np.float32)
    toks = np.zeros((8, D), np.int32)
    ua = np.zeros((8, D), np.float32)
    us = np.full(8, 0.6, np.float32)
    P[:] = 1.0 / V
    Q[:] = 1.0 / V
    P[0, 0] = 0.5 / V                       # p <= q everywhere: empty residual after rejection
    ua[0, 0] = 0.9
    P[1, 0] = 0.0                           # all-zero: reject, empty residual, empty fallback
    toks[2, 1] = 99                         # out-of-range token at draft 2
    Q[3, 0, 2] = np.nan                     # NaN at the tested token
    toks[3, 0] = 2
    P[4, 0] = 0.0
    P[4, 0, 5] = 1.0                        # one-hot target: always reject, yields 5
    Q[5, 0] = 0.0
    Q[5, 0, 1] = 1.0                        # one-hot draft
    toks[5, 0] = 1
    ua[5, 0] = 0.5
    us[6] = 0.0                             # smallest uniform
    us[7] = np.float32(1 - 2.0 ** -24)      # largest uniform
    k = np.array([4, 4, 4, 4, 4, 4, 1, 4])
    qo = np.concatenate([[0], np.cumsum(k)]).astype(np.int32)
    target = np.concatenate([P[i, :k[i]] for i in range(8)])
    g = gpu_accept(dev, target, Q, toks, qo, ua, us, "probs", "f32")
    o = orc.accept(target, Q, toks, qo, ua, us, kind="probs")
    assert_exact(g, o)
    assert g["flags"][0] == 1 and g["flags"][1] == 3 and g["flags"][2] & 4


def test_all_positions_pruned(dev, orc):
    """K = R: every request keeps only its certain position (plain decode step)."""
    rng = np.random.default_rng(3)
    R, b, V = 50, 16, 5000
    qo = np.arange(R + 1, dtype=np.int32)
    target = _rand_rows(rng, R, V)
    draft = _rand_rows(rng, R * (b - 1), V).reshape(R, b - 1, V)
    toks = rng.integers(0, V, size=(R, b - 1)).astype(np.int32)
    ua = rng.random((R, b - 1)).astype(np.float32)
    us = (rng.integers(0, 1 << 24, size=R) * 2.0 ** -24).astype(np.float32)
    g = gpu_accept(dev, target, draft, toks, qo, ua, us, "probs", "f32")
    o = orc.accept(target, draft, toks, qo, ua, us, kind="probs")
    assert_exact(g, o)
    assert np.all(g["accept_len"] == 0) and np.all(g["out_tokens"][:, 1:] == -1)


def test_repeatable_bitwise(dev):
    cfg_name = "c16_b16"
    cfg, target, draft, toks, qo, ua, us, dtype = _workload(cfg_name, "logits")
    a, b = gpu_accept(dev, target, draft, toks, qo, ua, us, "logits", dtype, repeat=2)
    assert_exact(a, b)


@pytest.mark.parametrize("name,fill", [("tiny", 0xFF), ("c64_b16", 0xFF), ("c64_b16", 0x01), ("sweep_mtp_c16", 0x7F)])
def test_workspace_contents_on_entry(dev, orc, name, fill):
    """Logits mode counts the draw's chunk workgroups on per-request arrival counters in the
    workspace, which the statistics pass zeroes first: whatever the workspace holds on
    entry (here every byte set to `fill`), the outputs equal the oracle's, and a second
    call on the same workspace gives the same outputs bit for bit."""
    from paper_2607_25852_amd import binding as B
    from paper_2607_25852_amd.round import to_dev
    say("accept workspace fill", name, hex(fill))
    cfg, target, draft, toks, qo, ua, us, dtype = _workload(name, "logits")
    target, draft = poisoned(target, draft, qo)
    R, D, V = draft.shape
    d = B.accept_desc(R, D + 1, V, B.SV_LOGITS, B.SV_F32 if dtype == "f32" else B.SV_BF16, 1.0)
    ws = dev.full((B.accept_workspace_size(d),), fill, dtype=dev.uint8, device="cuda")
    tg, dr = to_dev(target), to_dev(draft)
    tk, qd = to_dev(np.ascontiguousarray(toks, np.int32)), to_dev(np.ascontiguousarray(qo, np.int32))
    uad, usd = to_dev(np.ascontiguousarray(ua, np.float32)), to_dev(np.ascontiguousarray(us, np.float32))
    outs = []
    for _ in range(2):
        acc = dev.full((R,), -9, dtype=dev.int32, device="cuda")
        out = dev.full((R, D + 1), -9, dtype=dev.int32, device="cuda")
        flags = dev.full((R,), -9, dtype=dev.int32, device="cuda")
        B.spec_accept(d, tg, dr, tk, qd, uad, usd, acc, out, flags, ws)
        dev.cuda.synchronize()
        outs.append(dict(accept_len=acc.cpu().numpy(), out_tokens=out.cpu().numpy(), flags=flags.cpu().numpy()))
    assert_exact(outs[1], outs[0])
    o = orc.accept(target[:int(qo[-1])], draft, toks, qo, ua, us, kind="logits", dtype=dtype, diagnostics=True)
    exact, marginal, failures = classify_accept(outs[0], o, ua)
    say("accept workspace fill", name, hex(fill), "exact", exact, "marginal", marginal, "fail", len(failures))
    assert not failures, failures[:5]
    assert marginal <= max(1, cfg.R // 50)


def test_many_requests_flat_grids(dev, orc):
    """70000 requests of block 2 (more row slots than one grid dimension holds):
    the flat grids of both kernels still cover every request, bit-exact in probs mode."""
    rng = np.random.default_rng(11)
    R, b, V = 70000, 2, 64
    target_full = _rand_rows(rng, R * b, V).reshape(R, b, V)
    draft = _rand_rows(rng, R * (b - 1), V).reshape(R, b - 1, V)
    k = rng.integers(1, b + 1, size=R)
    from paper_2607_25852_amd import synth
    qo = synth.indptr_from_depths(k.astype(np.int32))
    target = np.concatenate([target_full[i, :k[i]] for i in range(R)])
    tokens = rng.integers(0, V, size=(R, b - 1)).astype(np.int32)
    ua = (rng.integers(0, 1 << 24, size=(R, b - 1)) * 2.0 ** -24).astype(np.float32)
    us = (rng.integers(0, 1 << 24, size=R) * 2.0 ** -24).astype(np.float32)
    say("accept many requests", R)
    g = gpu_accept(dev, target, draft, tokens, qo, ua, us, "probs", "f32")
    o = orc.accept(target, draft, tokens, qo, ua, us, kind="probs", dtype="f32")
    assert_exact(g, o)


def test_many_requests_flat_grids_logits(dev, orc):
    """Logits mode at 40000 requests of block 3: the statistics pass covers 200000 row
    slots on one flat grid."""
    rng = np.random.default_rng(12)
    R, b, V = 40000, 3, 96
    D = b - 1
    k = rng.integers(1, b + 1, size=R)
    from paper_2607_25852_amd import synth
    qo = synth.indptr_from_depths(k.astype(np.int32))
    tl = (rng.standard_normal((int(qo[-1]), V)) * 2).astype(np.float32)
    dl = (rng.standard_normal((R, D, V)) * 2).astype(np.float32)
    toks = rng.integers(0, V, size=(R, D)).astype(np.int32)
    ua = (rng.integers(0, 1 << 24, size=(R, D)) * 2.0 ** -24).astype(np.float32)
    us = (rng.integers(0, 1 << 24, size=R) * 2.0 ** -24).astype(np.float32)
    say("accept many requests logits", R)
    g = gpu_accept(dev, tl, dl, toks, qo, ua, us, "logits", "f32")
    o = orc.accept(tl, dl, toks, qo, ua, us, kind="logits", dtype="f32", diagnostics=True)
    exact, marginal, failures = classify_accept(g, o, ua)
    assert not failures, failures[:5]
    assert marginal <= 3


def _greedy_tokens(rng, target_f32, qo, D, share=0.75):
    """draft tokens: the argmax of the target row with probability `share`, else random"""
    R = len(qo) - 1
    V = target_f32.shape[1]
    tok = rng.integers(0, V, size=(R, D)).astype(np.int32)
    for i in range(R):
        for t in range(int(qo[i + 1] - qo[i]) - 1):
            row = target_f32[qo[i] + t]
            if rng.random() < share and not np.all(np.isnan(row)):
                tok[i, t] = int(np.nanargmax(row))
    return tok


def gpu_greedy(torch, target, D, tokens, qo, kind, dtype):
    """greedy call with NULL draft rows and uniforms (they are not read)"""
    from paper_2607_25852_amd import binding as B
    from paper_2607_25852_amd.round import to_dev
    R, V = len(qo) - 1, target.shape[1]
    b = D + 1
    d = B.accept_desc(R, b, V, B.SV_PROBS if kind == "probs" else B.SV_LOGITS,
                      B.SV_F32 if dtype == "f32" else B.SV_BF16, 0.0)
    ws = torch.empty(B.accept_workspace_size(d), dtype=torch.uint8, device="cuda")
    acc = torch.full((R,), -9, dtype=torch.int32, device="cuda")
    out = torch.full((R, b), -9, dtype=torch.int32, device="cuda")
    flags = torch.full((R,), -9, dtype=torch.int32, device="cuda")
    B.spec_accept(d, to_dev(target), None, to_dev(np.ascontiguousarray(tokens, np.int32)),
                  to_dev(np.ascontiguousarray(qo, np.int32)), None, None, acc, out, flags, ws)
    torch.cuda.synchronize()
    return dict(accept_len=acc.cpu().numpy(), out_tokens=out.cpu().numpy(), flags=flags.cpu().numpy())


@pytest.mark.parametrize("name", ["tiny", "c16_b16", "c64_b16", "sweep_mtp_c32"])
def test_greedy_logits_bit_exact(dev, orc, name):
    """temperature 0 on the workload's logits: argmax decisions are exact on both sides"""
    from paper_2607_25852_amd import synth
    cfg, target, draft, _, qo, _, _, dtype = _workload(name, "logits")
    tf = synth.bf16_to_f32(target) if dtype == "bf16" else target
    tokens = _greedy_tokens(np.random.default_rng(5), tf, qo, cfg.D, share=0.9)
    say("accept greedy", name)
    g = gpu_greedy(dev, target, cfg.D, tokens, qo, "logits", dtype)
    o = orc.accept_greedy(target, (cfg.R, cfg.D, cfg.V), tokens, qo, dtype=dtype)
    assert_exact(g, o)
    assert np.mean(o["accept_len"]) > 1.0  # long accepted prefixes were exercised


@pytest.mark.parametrize("V", [1, 7, 1000, 8192, 16385, 40000])
def test_greedy_ties_nan_ragged(dev, orc, V):
    """coarse values (many ties), NaN entries, an all-NaN row, out-of-range tokens,
    ragged vocabulary sizes; fp32 logits, bf16 logits and fp32 probabilities"""
    from paper_2607_25852_amd import synth
    rng = np.random.default_rng(V)
    R, b = 19, 7
    D = b - 1
    k = rng.integers(1, b + 1, size=R)
    qo = synth.indptr_from_depths(k.astype(np.int32))
    x = rng.integers(-3, 4, size=(int(qo[-1]), V)).astype(np.float32)
    x[rng.random(x.shape) < 0.05] = np.nan
    x[int(qo[3])] = np.nan  # a whole row
    tokens = _greedy_tokens(rng, x, qo, D)
    tokens[2, 0] = V + 3
    tokens[5, 0] = -1
    for kind, dtype, tgt in [("logits", "f32", x), ("logits", "bf16", synth.bf16_bits(x)), ("probs", "f32", x)]:
        g = gpu_greedy(dev, tgt, D, tokens, qo, kind, dtype)
        o = orc.accept_greedy(tgt, (R, D, V), tokens, qo, dtype=dtype)
        assert_exact(g, o)


def test_large_shape_without_partials(dev, orc):
    """16400 requests over a 8193-token vocabulary: the per-thread partial sums would exceed
    their 64 MB cap (16400 x 2 chunks x 256 threads x 8 B), so the draw searches its chunk
    by rescanning it. The last chunk holds a single token. Bit-exact in probs mode."""
    rng = np.random.default_rng(13)
    R, b, V = 16400, 2, 8193
    assert R * ((V + 8191) // 8192) * 256 * 8 > 64 << 20
    k = rng.integers(1, b + 1, size=R)
    from paper_2607_25852_amd import synth
    qo = synth.indptr_from_depths(k.astype(np.int32))
    # uniform rows scaled to sum to about 1 (exact normalisation is not needed for parity)
    target = rng.random((int(qo[-1]), V), dtype=np.float32)
    target *= np.float32(2.0 / V)
    draft = rng.random((R, b - 1, V), dtype=np.float32)
    draft *= np.float32(2.0 / V)
    tokens = rng.integers(0, V, size=(R, b - 1)).astype(np.int32)
    ua = (rng.integers(0, 1 << 24, size=(R, b - 1)) * 2.0 ** -24).astype(np.float32)
    us = (rng.integers(0, 1 << 24, size=R) * 2.0 ** -24).astype(np.float32)
    say("accept without partials", R, V)
    g = gpu_accept(dev, target, draft, tokens, qo, ua, us, "probs", "f32")
    o = orc.accept(target, draft, tokens, qo, ua, us, kind="probs", dtype="f32")
    assert_exact(g, o)
    assert np.any(g["out_tokens"][:, :] >= 8192)  # some draws land in the one-token chunk


def test_largest_vocabulary_logits(dev, orc):
    """bf16 logits over the largest vocabulary the library accepts (2^22 tokens: 512
    residual chunks and 256 statistics chunks per row), ragged blocks of up to 4."""
    from paper_2607_25852_amd import synth
    rng = np.random.default_rng(14)
    R, b, V = 3, 4, 1 << 22
    D = b - 1
    k = np.array([4, 1, 3], dtype=np.int32)
    qo = synth.indptr_from_depths(k)
    tl = (rng.standard_normal((int(qo[-1]), V), dtype=np.float32) * 4).astype(np.float32)
    dl = (rng.standard_normal((R, D, V), dtype=np.float32) * 4).astype(np.float32)
    for i in range(R):  # drafts close to their target rows, except request 2's second draft
        n = k[i] - 1
        dl[i, :n] = tl[qo[i]:qo[i] + n] + rng.standard_normal((n, V), dtype=np.float32)
    tl, dl = synth.bf16_bits(tl), synth.bf16_bits(dl)
    toks = np.stack([[int(np.argmax(dl[i, t])) if t % 2 == 0 else int(rng.integers(0, V)) for t in range(D)]
                     for i in range(R)]).astype(np.int32)
    # the drafted token's target logit far below its draft logit: rejected, residual draw
    toks[2, 1] = int(np.argmin(synth.bf16_to_f32(tl[qo[2] + 1]) - synth.bf16_to_f32(dl[2, 1])))
    ua = (rng.integers(0, 1 << 24, size=(R, D)) * 2.0 ** -24).astype(np.float32)
    us = (rng.integers(0, 1 << 24, size=R) * 2.0 ** -24).astype(np.float32)
    say("accept largest vocabulary", V)
    g = gpu_accept(dev, tl, dl, toks, qo, ua, us, "logits", "bf16", 1.0)
    o = orc.accept(tl, dl, toks, qo, ua, us, kind="logits", dtype="bf16", temperature=1.0, diagnostics=True)
    exact, marginal, failures = classify_accept(g, o, ua)
    assert not failures, failures[:5]
    assert marginal <= 1


# ------------------------------------------------------------------------------------
# Replay of logits-mode decisions: the kernel's own fp32 values, handed to the oracle's
# probability-mode procedure, must reproduce every output bit for bit.
# ------------------------------------------------------------------------------------
def gpu_accept_debug(torch, target, draft, tokens, qo, ua, us, dtype, T=1.0):
    from paper_2607_25852_amd import binding as B
    from paper_2607_25852_amd.round import to_dev
    R, D, V = draft.shape
    b = D + 1
    d = B.accept_desc(R, b, V, B.SV_LOGITS, B.SV_F32 if dtype == "f32" else B.SV_BF16, T)
    ws = torch.empty(B.accept_workspace_size(d), dtype=torch.uint8, device="cuda")
    acc = torch.full((R,), -9, dtype=torch.int32, device="cuda")
    out = torch.full((R, b), -9, dtype=torch.int32, device="cuda")
    flags = torch.full((R,), -9, dtype=torch.int32, device="cuda")
    dpq = torch.full((2, R, max(D, 1)), float("nan"), dtype=torch.float32, device="cuda")
    drow = torch.full((R, 2, V), float("nan"), dtype=torch.float32, device="cuda")
    B.spec_accept_debug(d, to_dev(target), to_dev(draft), to_dev(np.ascontiguousarray(tokens, np.int32)),
                        to_dev(np.ascontiguousarray(qo, np.int32)), to_dev(np.ascontiguousarray(ua, np.float32)),
                        to_dev(np.ascontiguousarray(us, np.float32)), acc, out, flags, dpq, drow, ws)
    torch.cuda.synchronize()
    g = dict(accept_len=acc.cpu().numpy(), out_tokens=out.cpu().numpy(), flags=flags.cpu().numpy())
    return g, dpq.cpu().numpy(), drow.cpu().numpy()


def replay_rows(g, dpq, drow, toks, qo, V):
    """Probability rows holding exactly what the kernel compared and weighed: P_{t-1}(d_t)
    and Q_t(d_t) at every tested token, and the full row pair of the draw."""
    R, D = toks.shape
    K = int(qo[-1])
    tgt = np.zeros((K, V), np.float32)
    dft = np.zeros((R, D, V), np.float32)
    for i in range(R):
        n = int(qo[i + 1] - qo[i]) - 1
        a = int(g["accept_len"][i])
        for t in range(n):
            d = int(toks[i, t])
            if 0 <= d < V:
                tgt[qo[i] + t, d] = dpq[0, i, t]
                dft[i, t, d] = dpq[1, i, t]
        tgt[qo[i] + a] = drow[i, 0]
        if a < n:
            dft[i, a] = drow[i, 1]
            d = int(toks[i, a])
            if 0 <= d < V:  # the draw's rows hold the very values the rejected test compared
                assert drow[i, 0, d].view(np.uint32) == dpq[0, i, a].view(np.uint32)
                assert drow[i, 1, d].view(np.uint32) == dpq[1, i, a].view(np.uint32)
    return tgt, dft


@pytest.mark.parametrize("name", ["tiny", "c16_b16", "c64_b16", "long_c32", "sweep_mtp_c8", "sweep_blk_c32"])
def test_logits_replay_bit_exact(dev, orc, name):
    say("accept replay", name)
    cfg, target, draft, toks, qo, ua, us, dtype = _workload(name, "logits")
    g, dpq, drow = gpu_accept_debug(dev, target, draft, toks, qo, ua, us, dtype)
    tgt, dft = replay_rows(g, dpq, drow, toks, qo, cfg.V)
    o = orc.accept(tgt, dft, toks, qo, ua, us, kind="probs")
    assert_exact(g, o)
    # the kernel's softmax values at the tested tokens against the oracle's fp64 ones
    ref = orc.accept(target, draft, toks, qo, ua, us, kind="logits", dtype=dtype, diagnostics=True)
    n = np.diff(qo) - 1
    # the tests the oracle evaluated: up to and including its first rejection
    last = np.minimum(ref["accept_len"], n - 1)
    mask = (np.arange(cfg.D)[None, :] <= last[:, None]) & (toks >= 0) & (toks < cfg.V)
    for got, want in ((dpq[0], ref["p_at"]), (dpq[1], ref["q_at"])):
        err = np.abs(got[mask].astype(np.float64) - want[mask])
        assert np.all(err <= 1e-6 + 1e-5 * np.abs(want[mask])), float(err.max())


@pytest.mark.parametrize("dtype,V,T", [("f32", 1000, 1.0), ("bf16", 4099, 0.6), ("bf16", 32768, 1.7)])
def test_logits_replay_ragged(dev, orc, dtype, V, T):
    from paper_2607_25852_amd import synth
    rng = np.random.default_rng(V + int(T * 10) + 5)
    R, b = 29, 11
    D = b - 1
    k = rng.integers(1, b + 1, size=R)
    qo = np.concatenate([[0], np.cumsum(k)]).astype(np.int32)
    tl = (rng.standard_normal((int(qo[-1]), V)) * 3).astype(np.float32)
    dl = (rng.standard_normal((R, D, V)) * 3).astype(np.float32)
    for i in range(R):
        n = k[i] - 1
        dl[i, :n] = tl[qo[i]:qo[i] + n] + rng.standard_normal((n, V)).astype(np.float32) * 0.7
    if dtype == "bf16":
        tl, dl = synth.bf16_bits(tl), synth.bf16_bits(dl)
    toks = rng.integers(0, V, size=(R, D)).astype(np.int32)
    toks[3, 0] = V + 5  # an out-of-range token is rejected (flag bit 2) on both sides
    ua = (rng.integers(0, 1 << 24, size=(R, D)) * 2.0 ** -24).astype(np.float32)
    us = (rng.integers(0, 1 << 24, size=R) * 2.0 ** -24).astype(np.float32)
    say("accept replay ragged", dtype, V, T)
    g, dpq, drow = gpu_accept_debug(dev, tl, dl, toks, qo, ua, us, dtype, T)
    tgt, dft = replay_rows(g, dpq, drow, toks, qo, V)
    o = orc.accept(tgt, dft, toks, qo, ua, us, kind="probs")
    assert_exact(g, o)
