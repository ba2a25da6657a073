"""Pins of the acceptance oracle against what rejection-sampling verification
must satisfy (Sec. 1: the committed tokens follow the target distribution;
eq. mtp-acceptance-tv: per-position acceptance equals the overlap sum_v min(p,q);
eq. mtp-e2e / eq. dcut-expected-progress: expected accepted length is the sum
of prefix products of the overlaps).

The central pin is exact: for small vocabularies the output distribution of each
committed position is enumerated over the whole 2^24 grid of both uniforms
(acceptance and the sampled token are monotone in their uniform, so binary
search finds every boundary) and must equal the target row of that position.
A dropped term, a wrong sign in the residual, or an off-by-one row index fails it.
"""
import numpy as np
import pytest
import scipy.special

GRID = 1 << 24


def _norm_f32(x):
    x = np.asarray(x, np.float64)
    return (x / x.sum(axis=-1, keepdims=True)).astype(np.float32)


def _pn(x):
    """fp64 normalised copy of a row (for drawing tokens with numpy)."""
    x = np.asarray(x, np.float64)
    return x / x.sum()


def _batch(P_rows, Q_rows, R):
    """Replicate one request's rows R times: P_rows [n+1, V], Q_rows [n, V]."""
    n = Q_rows.shape[0]
    V = P_rows.shape[1]
    target = np.tile(P_rows[None], (R, 1, 1)).reshape(R * (n + 1), V)
    draft = np.zeros((R, max(n, 1), V), np.float32)
    if n:
        draft[:, :n] = Q_rows[None]
    qo = np.arange(R + 1, dtype=np.int32) * (n + 1)
    return target, draft, qo


def _run(orc, target, draft, qo, toks, ua, us):
    return orc.accept(target, draft, toks, qo, ua, us, kind="probs")


def _search(pred_fn, R):
    """Smallest m in [0, GRID] with pred(m) true per request (pred monotone false->true)."""
    lo = np.zeros(R, np.int64)
    hi = np.full(R, GRID, np.int64)
    while np.any(lo < hi):
        mid = (lo + hi) // 2
        ok = pred_fn(np.minimum(mid, GRID - 1)) & (mid < GRID)
        hi = np.where(ok, mid, hi)
        lo = np.where(ok, lo, mid + 1)
    return lo


def _position_distribution(orc, P_rows, Q_rows, t):
    """Exact distribution of the token committed at block position t (1-based),
    given that drafts 1..t-1 were accepted. Drafts before t are fixed to token 0
    with u = 0 (accepted since P > 0); draft t ranges over every x with weight Q_t(x).
    t = n+1 means the bonus position (every draft accepted)."""
    n = Q_rows.shape[0]
    V = P_rows.shape[1]
    D = max(n, 1)
    if t == n + 1:  # bonus: sampled from P_n by u_sample only
        R = V
        target, draft, qo = _batch(P_rows, Q_rows, R)
        toks = np.zeros((R, D), np.int32)
        ua = np.zeros((R, D), np.float32)
        ys = np.arange(V)

        def tok_ge(m):
            r = _run(orc, target, draft, qo, toks, ua, (m * 2.0 ** -24).astype(np.float32))
            assert np.all(r["accept_len"] == n)
            return r["out_tokens"][:, n] >= ys

        B = _search(tok_ge, R)
        cnt = np.diff(np.append(B, GRID))
        return cnt / GRID
    # acceptance counts for each draft token x at position t
    R = V
    target, draft, qo = _batch(P_rows, Q_rows, R)
    xs = np.arange(V)
    toks = np.zeros((R, D), np.int32)
    toks[:, t - 1] = xs

    def rejects(m):
        ua = np.zeros((R, D), np.float32)
        ua[:, t - 1] = (m * 2.0 ** -24).astype(np.float32)
        r = _run(orc, target, draft, qo, toks, ua, np.zeros(R, np.float32))
        assert np.all(r["accept_len"] >= t - 1)
        return r["accept_len"] == t - 1

    acc = _search(rejects, R)  # number of accepting grid points per x
    # residual sample after rejecting x at position t: intervals of u_sample
    R2 = V * V
    target, draft, qo = _batch(P_rows, Q_rows, R2)
    xx = np.repeat(xs, V)
    yy = np.tile(xs, V)
    toks = np.zeros((R2, D), np.int32)
    toks[:, t - 1] = xx
    ua = np.zeros((R2, D), np.float32)
    ua[:, t - 1] = np.float32(1.0 - 2.0 ** -24)

    def tok_ge(m):
        r = _run(orc, target, draft, qo, toks, ua, (m * 2.0 ** -24).astype(np.float32))
        return r["out_tokens"][:, t - 1] >= yy

    B = _search(tok_ge, R2).reshape(V, V)
    cnt = np.diff(np.concatenate([B, np.full((V, 1), GRID)], axis=1), axis=1)
    res = cnt / GRID  # [x, y]
    q = Q_rows[t - 1].astype(np.float64)
    q = q / q.sum()
    a = acc / GRID
    dist = (q * a) @ np.eye(V) + ((q * (1 - a))[:, None] * res).sum(axis=0)
    # rejection never happens for x where acc == GRID: its residual row is irrelevant
    return dist


@pytest.mark.parametrize("V,n,seed", [(5, 1, 0), (8, 1, 1), (6, 2, 2), (7, 3, 3)])
def test_output_distribution_equals_target_exactly(orc, V, n, seed):
    rng = np.random.default_rng(seed)
    P = _norm_f32(rng.gamma(0.7, size=(n + 1, V)) + 0.02)
    Q = _norm_f32(rng.gamma(0.7, size=(n, V)) + 0.02)
    tol = 4 * V * 2.0 ** -24 + 1e-9
    for t in range(1, n + 2):
        dist = _position_distribution(orc, P, Q, t)
        want = _pn(P[t - 1])
        np.testing.assert_allclose(dist, want, atol=tol, rtol=0)
        assert abs(dist.sum() - 1.0) < 1e-12


def test_identity_fails_for_a_planted_mistake(orc):
    """Guard on the pin itself: a wrong-row test (draft t judged against P_t
    instead of P_{t-1}) breaks the identity by far more than the tolerance."""
    rng = np.random.default_rng(11)
    V = 6
    P = _norm_f32(rng.gamma(0.7, size=(3, V)) + 0.02)
    Q = _norm_f32(rng.gamma(0.7, size=(2, V)) + 0.02)
    dist = _position_distribution(orc, P[1:], Q[1:], 1)  # rows shifted by one
    want = _pn(P[0])
    assert np.abs(dist - want).max() > 1e-3


def test_overlap_is_acceptance_rate(orc):
    """eq. mtp-acceptance-tv: Pr(accept) = sum_v min(p, q) = 1 - TV(p, q)."""
    rng = np.random.default_rng(5)
    V, R = 16, 200000
    P = _norm_f32(rng.gamma(0.5, size=(2, V)))
    Q = _norm_f32(rng.gamma(0.5, size=(1, V)))
    target, draft, qo = _batch(P, Q, R)
    q = _pn(Q[0])
    toks = rng.choice(V, size=(R, 1), p=q).astype(np.int32)
    ua = (rng.integers(0, GRID, size=(R, 1)) * 2.0 ** -24).astype(np.float32)
    us = (rng.integers(0, GRID, size=R) * 2.0 ** -24).astype(np.float32)
    r = orc.accept(target, draft, toks, qo, ua, us, kind="probs")
    rate = (r["accept_len"] == 1).mean()
    alpha = np.minimum(P[0].astype(np.float64), Q[0].astype(np.float64)).sum()
    tv = 0.5 * np.abs(P[0].astype(np.float64) - Q[0].astype(np.float64)).sum()
    assert abs(alpha - (1 - tv)) < 1e-6
    sigma = np.sqrt(alpha * (1 - alpha) / R)
    assert abs(rate - alpha) < 4 * sigma


def test_expected_accepted_length(orc):
    """With identical rows at every position, E[a] = sum_{m=1..n} alpha^m
    (the prefix-product sum of eq. mtp-e2e / eq. dcut-expected-progress)."""
    rng = np.random.default_rng(6)
    V, n, R = 12, 4, 100000
    p = _norm_f32(rng.gamma(0.6, size=V))
    qd = _norm_f32(rng.gamma(0.6, size=V))
    P = np.tile(p, (n + 1, 1))
    Q = np.tile(qd, (n, 1))
    target, draft, qo = _batch(P, Q, R)
    q64 = _pn(qd)
    toks = rng.choice(V, size=(R, n), p=q64).astype(np.int32)
    ua = (rng.integers(0, GRID, size=(R, n)) * 2.0 ** -24).astype(np.float32)
    us = (rng.integers(0, GRID, size=R) * 2.0 ** -24).astype(np.float32)
    r = orc.accept(target, draft, toks, qo, ua, us, kind="probs")
    a = r["accept_len"].astype(np.float64)
    alpha = np.minimum(p.astype(np.float64), qd.astype(np.float64)).sum()
    want = sum(alpha ** m for m in range(1, n + 1))
    assert abs(a.mean() - want) < 4 * a.std() / np.sqrt(R)
    # committed count is a + 1; tokens past the cut are -1
    out = r["out_tokens"]
    for i in range(50):
        ai = int(r["accept_len"][i])
        assert np.all(out[i, :ai] == toks[i, :ai]) and out[i, ai] >= 0 and np.all(out[i, ai + 1:] == -1)


def test_identical_distributions_accept_everything(orc):
    rng = np.random.default_rng(8)
    V, n, R = 32, 5, 2000
    rows = _norm_f32(rng.gamma(0.5, size=(n + 1, V)) + 1e-3)
    target, draft, qo = _batch(rows, rows[:n], R)
    toks = np.stack([rng.choice(V, size=R, p=_pn(rows[t]))
                     for t in range(n)], axis=1).astype(np.int32)
    ua = (rng.integers(0, GRID, size=(R, n)) * 2.0 ** -24).astype(np.float32)
    us = (rng.integers(0, GRID, size=R) * 2.0 ** -24).astype(np.float32)
    r = orc.accept(target, draft, toks, qo, ua, us, kind="probs")
    assert np.all(r["accept_len"] == n)
    assert np.all(r["out_tokens"][:, :n] == toks)


def test_bonus_distribution_is_last_row(orc):
    rng = np.random.default_rng(9)
    V = 9
    P = _norm_f32(rng.gamma(0.8, size=(3, V)) + 0.01)
    dist = _position_distribution(orc, P, P[:2], 3)
    np.testing.assert_allclose(dist, _pn(P[2]), atol=4 * V * 2.0 ** -24)


def test_one_hot_draft(orc):
    """q = delta_d: accepted iff u < p(d) (exactly ceil(p(d) 2^24) grid points);
    the residual is p without d, renormalised."""
    rng = np.random.default_rng(10)
    V, d = 7, 3
    P = _norm_f32(rng.gamma(1.0, size=(2, V)) + 0.05)
    Q = np.zeros((1, V), np.float32)
    Q[0, d] = 1.0
    target, draft, qo = _batch(P, Q, 1)
    toks = np.array([[d]], np.int32)

    def rejects(m):
        r = _run(orc, target, draft, qo, toks, (m * 2.0 ** -24).astype(np.float32).reshape(1, 1),
                 np.zeros(1, np.float32))
        return r["accept_len"] == 0

    acc = _search(rejects, 1)[0]
    assert acc == int(np.ceil(np.float64(P[0, d]) * GRID))
    dist = _position_distribution(orc, P, Q, 1)
    np.testing.assert_allclose(dist, _pn(P[0]), atol=4 * V * 2.0 ** -24)
    # residual alone
    r = _run(orc, np.tile(target, (1, 1)), draft, qo, toks, np.full((1, 1), 1 - 2.0 ** -24, np.float32),
             np.array([0.0], np.float32))
    assert r["out_tokens"][0, 0] != d


def test_one_hot_target_always_rejects_and_yields_its_token(orc):
    rng = np.random.default_rng(12)
    V, y = 10, 6
    P = np.zeros((2, V), np.float32)
    P[0, y] = 1.0
    P[1] = _norm_f32(rng.random(V))
    Q = _norm_f32(rng.random((1, V)) + 0.1)
    R = 500
    target, draft, qo = _batch(P, Q, R)
    toks = rng.choice([v for v in range(V) if v != y], size=(R, 1)).astype(np.int32)
    ua = (rng.integers(0, GRID, size=(R, 1)) * 2.0 ** -24).astype(np.float32)
    us = (rng.integers(0, GRID, size=R) * 2.0 ** -24).astype(np.float32)
    r = orc.accept(target, draft, toks, qo, ua, us, kind="probs")
    assert np.all(r["accept_len"] == 0) and np.all(r["out_tokens"][:, 0] == y)


def test_no_drafts_is_a_plain_decode_step(orc):
    rng = np.random.default_rng(13)
    V = 8
    P = _norm_f32(rng.random((1, V)) + 0.05)
    dist = _position_distribution(orc, P, np.zeros((0, V), np.float32), 1)
    np.testing.assert_allclose(dist, _pn(P[0]), atol=4 * V * 2.0 ** -24)


def test_zero_uniform_accepts_iff_target_positive(orc):
    V = 4
    P = np.array([[0.0, 0.5, 0.5, 0.0], [0.25, 0.25, 0.25, 0.25]], np.float32)
    Q = np.array([[0.25, 0.25, 0.25, 0.25]], np.float32)
    target, draft, qo = _batch(P, Q, 4)
    toks = np.arange(4, dtype=np.int32).reshape(4, 1)
    r = orc.accept(target, draft, toks, qo, np.zeros((4, 1), np.float32), np.zeros(4, np.float32))
    np.testing.assert_array_equal(r["accept_len"], [0, 1, 1, 0])


def test_degenerate_rows_and_flags(orc):
    V = 4
    # rejection with an empty residual (p <= q everywhere): falls back to p, flag bit 0
    P = np.array([[0.1, 0.1, 0.1, 0.1], [0.25] * 4], np.float32)
    Q = np.array([[0.25, 0.25, 0.25, 0.25]], np.float32)
    target, draft, qo = _batch(P, Q, 1)
    r = orc.accept(target, draft, np.array([[2]], np.int32), qo, np.full((1, 1), 0.9, np.float32),
                   np.array([0.6], np.float32))
    assert r["accept_len"][0] == 0 and r["flags"][0] == 1 and r["out_tokens"][0, 0] == 2
    # all-zero target row: no token can be drawn, flag bits 0 and 1
    P = np.zeros((2, V), np.float32)
    target, draft, qo = _batch(P, Q, 1)
    r = orc.accept(target, draft, np.array([[2]], np.int32), qo, np.zeros((1, 1), np.float32),
                   np.array([0.6], np.float32))
    assert r["accept_len"][0] == 0 and r["flags"][0] == 3 and r["out_tokens"][0, 0] == -1
    # a draft token outside the vocabulary is rejected, flag bit 2
    P = np.array([[0.25] * 4, [0.25] * 4], np.float32)
    Q = np.array([[0.5, 0.5, 0.0, 0.0]], np.float32)
    target, draft, qo = _batch(P, Q, 1)
    r = orc.accept(target, draft, np.array([[9]], np.int32), qo, np.zeros((1, 1), np.float32),
                   np.array([0.0], np.float32))
    assert r["accept_len"][0] == 0 and r["flags"][0] & 4
    # NaN in the draft row at the tested token rejects
    Q = np.array([[np.nan, 0.5, 0.25, 0.25]], np.float32)
    target, draft, qo = _batch(P, Q, 1)
    r = orc.accept(target, draft, np.array([[0]], np.int32), qo, np.zeros((1, 1), np.float32),
                   np.array([0.0], np.float32))
    assert r["accept_len"][0] == 0


def test_ragged_batch_matches_requests_run_alone(orc):
    rng = np.random.default_rng(14)
    V, b, R = 50, 6, 12
    D = b - 1
    k = rng.integers(1, b + 1, size=R)
    qo = np.zeros(R + 1, np.int32)
    qo[1:] = np.cumsum(k)
    target = _norm_f32(rng.gamma(0.5, size=(qo[-1], V)) + 1e-4)
    draft = _norm_f32(rng.gamma(0.5, size=(R, D, V)) + 1e-4)
    toks = rng.integers(0, V, size=(R, D)).astype(np.int32)
    ua = (rng.integers(0, GRID, size=(R, D)) * 2.0 ** -24).astype(np.float32)
    us = (rng.integers(0, GRID, size=R) * 2.0 ** -24).astype(np.float32)
    full = orc.accept(target, draft, toks, qo, ua, us)
    for i in range(R):
        one = orc.accept(target[qo[i]:qo[i + 1]], draft[i:i + 1], toks[i:i + 1],
                         np.array([0, k[i]], np.int32), ua[i:i + 1], us[i:i + 1])
        assert one["accept_len"][0] == full["accept_len"][i]
        np.testing.assert_array_equal(one["out_tokens"][0], full["out_tokens"][i])
        assert full["accept_len"][i] <= k[i] - 1


@pytest.mark.parametrize("dtype,T", [("f32", 1.0), ("bf16", 1.0), ("f32", 0.7)])
def test_logits_mode_is_library_softmax_then_probs_mode(orc, dtype, T):
    """Logits mode = softmax(l/T) (library routine, fp64) rounded to fp32, then the
    probability-mode procedure."""
    from paper_2607_25852_amd import synth
    rng = np.random.default_rng(15)
    V, b, R = 300, 5, 40
    D = b - 1
    qo = np.arange(R + 1, dtype=np.int32) * b
    tl = (rng.standard_normal((R * b, V)) * 2.5).astype(np.float32)
    dl = (tl.reshape(R, b, V)[:, :D] + rng.standard_normal((R, D, V)) * 0.7).astype(np.float32)
    if dtype == "bf16":
        tst, dst = synth.bf16_bits(tl), synth.bf16_bits(dl)
        tl, dl = synth.bf16_to_f32(tst), synth.bf16_to_f32(dst)
    else:
        tst, dst = tl, dl
    x_t = (tl / np.float32(T)).astype(np.float64)
    x_d = (dl / np.float32(T)).astype(np.float64)
    tp = scipy.special.softmax(x_t, axis=-1).astype(np.float32)
    dp = scipy.special.softmax(x_d, axis=-1).astype(np.float32)
    toks = np.stack([[rng.choice(V, p=_pn(dp[i, t])) for t in range(D)]
                     for i in range(R)]).astype(np.int32)
    ua = (rng.integers(0, GRID, size=(R, D)) * 2.0 ** -24).astype(np.float32)
    us = (rng.integers(0, GRID, size=R) * 2.0 ** -24).astype(np.float32)
    lg = orc.accept(tst, dst, toks, qo, ua, us, kind="logits", dtype=dtype, temperature=T, diagnostics=True)
    pr = orc.accept(tp, dp, toks, qo, ua, us, kind="probs", diagnostics=True)
    ulp = np.spacing(np.abs(pr["p_at"]).astype(np.float32)).astype(np.float64)
    assert np.all(np.abs(lg["p_at"] - pr["p_at"]) <= ulp)
    assert np.all(np.abs(lg["q_at"] - pr["q_at"]) <= np.spacing(np.abs(pr["q_at"]).astype(np.float32)))
    np.testing.assert_array_equal(lg["accept_len"], pr["accept_len"])
    np.testing.assert_array_equal(lg["out_tokens"], pr["out_tokens"])
