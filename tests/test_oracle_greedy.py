"""Pins of the oracle's greedy verification (temperature 0).

Greedy verification is rejection sampling with one-hot target and draft rows: with
p' = onehot(argmax P) and q' = onehot(d_t), the acceptance test u*q'(d) < p'(d) holds iff
d == argmax P, the residual after a rejection is onehot(argmax P), and the bonus row is
onehot(argmax P_n). The sampling path of the oracle (pinned separately by exact
enumeration) must therefore reproduce the greedy path for any uniforms.
"""
import numpy as np
import pytest

import oracle
from paper_2607_25852_amd import synth


def _onehot_rows(x):
    """fp32 one-hot rows at the argmax (NaN skipped, lowest index); an all-NaN row stays zero."""
    out = np.zeros(x.shape, np.float32)
    flat = x.reshape(-1, x.shape[-1])
    o = out.reshape(-1, x.shape[-1])
    for r in range(flat.shape[0]):
        if not np.all(np.isnan(flat[r])):
            o[r, np.nanargmax(flat[r])] = 1.0
    return out


@pytest.mark.parametrize("seed", range(6))
def test_greedy_equals_sampling_with_one_hot_rows(seed):
    rng = np.random.default_rng(seed)
    R, b, V = 13, 9, 37
    D = b - 1
    k = rng.integers(1, b + 1, size=R)
    qo = synth.indptr_from_depths(k.astype(np.int32))
    # coarse values so ties are common
    target = rng.integers(0, 6, size=(int(qo[-1]), V)).astype(np.float32)
    tokens = rng.integers(0, V, size=(R, D)).astype(np.int32)
    # make a good share of drafts correct so long accepted prefixes occur
    for i in range(R):
        for t in range(k[i] - 1):
            if rng.random() < 0.7:
                tokens[i, t] = int(np.nanargmax(target[qo[i] + t]))
    g = oracle.accept_greedy(target, (R, D, V), tokens, qo)
    p1 = _onehot_rows(target)
    q1 = np.zeros((R, D, V), np.float32)
    for i in range(R):
        for t in range(D):
            q1[i, t, tokens[i, t]] = 1.0
    for _ in range(3):
        ua = (rng.integers(0, 1 << 24, size=(R, D)) * 2.0 ** -24).astype(np.float32)
        us = (rng.integers(0, 1 << 24, size=R) * 2.0 ** -24).astype(np.float32)
        s = oracle.accept(p1, q1, tokens, qo, ua, us, kind="probs")
        np.testing.assert_array_equal(g["accept_len"], s["accept_len"])
        np.testing.assert_array_equal(g["out_tokens"], s["out_tokens"])
        np.testing.assert_array_equal(g["flags"], s["flags"])


def test_greedy_hand_cases():
    V = 5
    nan = np.nan
    target = np.array([
        [1, 3, 3, 0, 2],      # request 0, P_0: tie 1/2 -> argmax 1
        [0, 0, 9, 9, 1],      # P_1: tie -> 2
        [5, 1, 1, 1, 1],      # P_2: 0
        [nan, 2, nan, 7, 7],  # request 1, P_0: NaN skipped, tie -> 3
        [nan] * 5,            # request 2, P_0: all NaN -> -1
        [1, 1, 1, 1, 1],      # request 3, P_0 (no drafts kept): all equal -> 0
    ], np.float32)
    qo = np.array([0, 3, 4, 5, 6], np.int32)
    tokens = np.array([[1, 2, 4], [3, 0, 0], [0, 0, 0], [7, 0, 0]], np.int32)
    r = oracle.accept_greedy(target, (4, 3, V), tokens, qo)
    # request 0: d1 = 1 = argmax P_0, d2 = 2 = argmax P_1, all kept -> bonus argmax P_2 = 0
    assert r["accept_len"].tolist() == [2, 0, 0, 0]
    assert r["out_tokens"][0].tolist() == [1, 2, 0, -1]
    # request 1: n = 0 -> token argmax P_0 = 3
    assert r["out_tokens"][1].tolist() == [3, -1, -1, -1]
    # request 2: all-NaN row -> no token, flag bit 1
    assert r["out_tokens"][2].tolist() == [-1, -1, -1, -1] and r["flags"][2] == 2
    assert r["out_tokens"][3].tolist() == [0, -1, -1, -1]
    assert r["flags"][[0, 1, 3]].tolist() == [0, 0, 0]
    # out-of-range draft token: rejected, flag bit 2, token = argmax P_0
    qo2 = np.array([0, 2], np.int32)
    r2 = oracle.accept_greedy(target[:2], (1, 3, V), np.array([[9, 2, 0]], np.int32), qo2)
    assert r2["accept_len"].tolist() == [0] and r2["out_tokens"][0].tolist() == [1, -1, -1, -1]
    assert r2["flags"].tolist() == [4]


def test_greedy_bf16_matches_nanargmax():
    rng = np.random.default_rng(3)
    R, b, V = 9, 6, 300
    k = rng.integers(1, b + 1, size=R)
    qo = synth.indptr_from_depths(k.astype(np.int32))
    x = (rng.standard_normal((int(qo[-1]), V)) * 2).astype(np.float32)
    bits = synth.bf16_bits(x)  # rounding creates ties
    xf = synth.bf16_to_f32(bits)
    tokens = np.zeros((R, b - 1), np.int32)
    for i in range(R):
        for t in range(k[i] - 1):
            tokens[i, t] = int(np.nanargmax(xf[qo[i] + t])) if t < 3 else 0
    r = oracle.accept_greedy(bits, (R, b - 1, V), tokens, qo, dtype="bf16")
    for i in range(R):
        n = k[i] - 1
        a = 0
        while a < n and tokens[i, a] == np.nanargmax(xf[qo[i] + a]):
            a += 1
        assert r["accept_len"][i] == a
        assert r["out_tokens"][i, a] == np.nanargmax(xf[qo[i] + a])
    # logits through the generic entry with temperature 0 take the greedy path
    r3 = oracle.accept(bits, np.zeros((R, b - 1, V), np.uint16), tokens, qo, np.zeros((R, b - 1), np.float32),
                       np.zeros(R, np.float32), kind="logits", dtype="bf16", temperature=0.0)
    np.testing.assert_array_equal(r3["out_tokens"], r["out_tokens"])
