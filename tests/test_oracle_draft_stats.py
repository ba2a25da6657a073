"""Pins of the oracle's draft-row statistics: the confidence equals the largest
probability of an independent softmax (scipy), closed forms for a uniform row and a row
with one raised logit, the temperature acting as a scale of the logits, bf16 decoding,
and agreement with the synthetic drafter's own confidences (computed by the input
generator from its sampling distribution)."""
import numpy as np
import scipy.special

import oracle
from paper_2607_25852_amd import synth


def test_conf_is_max_softmax():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal((7, 3, 500)) * 3).astype(np.float32)
    st = oracle.draft_stats(x)
    p = scipy.special.softmax(x.astype(np.float64), axis=-1)
    np.testing.assert_allclose(st["conf"], p.max(axis=-1), rtol=1e-12)
    np.testing.assert_array_equal(st["m"], x.max(axis=-1).astype(np.float64))


def test_closed_forms():
    V = 4096
    st = oracle.draft_stats(np.full((1, V), 2.5, np.float32))
    assert st["S"][0] == V and st["conf"][0] == 1.0 / V
    L = 6.0
    x = np.zeros((1, V), np.float32)
    x[0, 17] = L
    st = oracle.draft_stats(x)
    np.testing.assert_allclose(st["conf"][0], 1.0 / (1.0 + (V - 1) * np.exp(-L)), rtol=1e-14)


def test_temperature_scales_logits():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((4, 300)).astype(np.float32)
    T = np.float32(0.5)  # a power of two: x / T is exact in fp32
    a = oracle.draft_stats(x, temperature=T)
    b = oracle.draft_stats((x / T).astype(np.float32))
    for k in ("m", "S", "conf"):
        np.testing.assert_allclose(a[k], b[k], rtol=1e-14)


def test_bf16_bits_decode():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((3, 64)).astype(np.float32)
    bits = synth.bf16_bits(x)
    a = oracle.draft_stats(bits, dtype="bf16")
    b = oracle.draft_stats(synth.bf16_to_f32(bits))
    for k in ("m", "S", "conf"):
        np.testing.assert_array_equal(a[k], b[k])


def test_matches_the_synthetic_drafter():
    cfg = synth.CONFIGS["tiny"]
    lr = synth.make_logits_round(cfg)
    st = oracle.draft_stats(lr["draft"], dtype=cfg.dtype)
    np.testing.assert_allclose(st["conf"], lr["conf"], rtol=2e-7)
