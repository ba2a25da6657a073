"""Pins of the verify-attention oracle by closed forms (no dense re-implementation):

* a single visible key returns its value row exactly; lse = its logit;
* two visible keys give the logistic weights sigma(z0 - z1);
* a zero query (or zero scale) weights every visible key equally, so with
  V_s = s the output is the mean visible position: this fixes the block-causal
  limit L_i + j exactly (row j of a block sees its own key and the ones before);
* head h reads kv-head floor(h / G) (grouped-query attention);
* a permuted page table (with pages moved accordingly) gives bit-identical
  results; NaN in pages and slots nobody may see never leaks;
* one dominant key returns its value row.
"""
import numpy as np
import pytest

from paper_2607_25852_amd import synth


def _cache_from_tokens(K_tok, V_tok, P, perm=None, fill=0.0):
    """Build [pages, Hkv, P, d] caches + page table for ONE request from per-token
    arrays [Hkv, n, d] (fp32)."""
    Hkv, n, d = K_tok.shape
    npg = -(-n // P)
    perm = np.arange(npg) if perm is None else perm
    kc = np.full((npg, Hkv, P, d), fill, np.float32)
    vc = np.full((npg, Hkv, P, d), fill, np.float32)
    for p in range(npg):
        lo, hi = p * P, min(n, (p + 1) * P)
        kc[perm[p], :, :hi - lo] = K_tok[:, lo:hi]
        vc[perm[p], :, :hi - lo] = V_tok[:, lo:hi]
    return kc, vc, perm.astype(np.int32)[None, :]


def test_single_key_returns_its_value(orc):
    rng = np.random.default_rng(0)
    d, Hq, Hkv = 16, 4, 2
    Kt = rng.standard_normal((Hkv, 1, d)).astype(np.float32)
    Vt = rng.standard_normal((Hkv, 1, d)).astype(np.float32)
    kc, vc, pt = _cache_from_tokens(Kt, Vt, 4)
    q = rng.standard_normal((1, Hq, d)).astype(np.float32)
    out, lse = orc.attention(q, kc, vc, pt, [0, 1], [1], scale=0.3)
    for h in range(Hq):
        np.testing.assert_array_equal(out[h], Vt[h // 2, 0].astype(np.float64))
        assert abs(lse[h] - 0.3 * np.dot(q[0, h].astype(np.float64), Kt[h // 2, 0])) < 1e-12


def test_two_keys_logistic(orc):
    rng = np.random.default_rng(1)
    d = 8
    Kt = rng.standard_normal((1, 2, d)).astype(np.float32)
    Vt = rng.standard_normal((1, 2, d)).astype(np.float32)
    kc, vc, pt = _cache_from_tokens(Kt, Vt, 16)
    q = rng.standard_normal((2, 1, d)).astype(np.float32)  # block of 2 rows, no context
    out, lse = orc.attention(q, kc, vc, pt, [0, 2], [2], scale=0.5)
    z = 0.5 * (Kt[0].astype(np.float64) @ q[1, 0].astype(np.float64))
    w0 = 1.0 / (1.0 + np.exp(z[1] - z[0]))
    np.testing.assert_allclose(out[1], w0 * Vt[0, 0] + (1 - w0) * Vt[0, 1], rtol=0, atol=1e-12)
    assert abs(lse[1] - np.logaddexp(z[0], z[1])) < 1e-12
    np.testing.assert_array_equal(out[0], Vt[0, 0].astype(np.float64))  # row 0 sees key 0 only


@pytest.mark.parametrize("L,k,P", [(0, 1, 16), (37, 8, 16), (128, 5, 16), (64, 16, 64), (3, 4, 2)])
def test_causal_limit_by_mean_position(orc, L, k, P):
    d, Hq, Hkv = 8, 6, 3
    n = L + k
    Kt = np.random.default_rng(2).standard_normal((Hkv, n, d)).astype(np.float32)
    Vt = np.broadcast_to(np.arange(n, dtype=np.float32)[None, :, None], (Hkv, n, d)).copy()
    kc, vc, pt = _cache_from_tokens(Kt, Vt, P, fill=np.nan)
    q = np.zeros((k, Hq, d), np.float32)
    out, lse = orc.attention(q, kc, vc, pt, [0, k], [n])
    out = out.reshape(k, Hq, d)
    lse = lse.reshape(k, Hq)
    for j in range(k):
        np.testing.assert_allclose(out[j], (L + j) / 2.0, rtol=0, atol=1e-9)
        np.testing.assert_allclose(lse[j], np.log(L + j + 1), rtol=0, atol=1e-12)


def test_grouped_query_head_map(orc):
    d, Hq, Hkv, n = 4, 8, 2, 5
    Kt = np.random.default_rng(3).standard_normal((Hkv, n, d)).astype(np.float32)
    Vt = np.zeros((Hkv, n, d), np.float32)
    Vt[1] = 1.0
    kc, vc, pt = _cache_from_tokens(Kt, Vt, 2)
    q = np.random.default_rng(4).standard_normal((1, Hq, d)).astype(np.float32)
    out, _ = orc.attention(q, kc, vc, pt, [0, 1], [n])
    np.testing.assert_allclose(out[:, 0], [0, 0, 0, 0, 1, 1, 1, 1], rtol=0, atol=1e-12)


def test_page_permutation_invariance_and_poison(orc):
    cfg = synth.CONFIGS["tiny"]
    L = synth.kv_context_lengths(cfg)
    k = np.array([8, 3, 1, 6], np.int32)
    qo = synth.indptr_from_depths(k)
    kv = synth.make_kv(cfg, L, fill_unused=np.nan)
    q = synth.pack_rows(kv["q_full"], qo)
    kvl = L + k
    out, lse = orc.attention(q, kv["k_cache"], kv["v_cache"], kv["page_table"], qo, kvl)
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(lse))
    # move every page to a new slot and relabel the table
    perm = np.random.default_rng(5).permutation(kv["num_pages"])
    kc2 = np.empty_like(kv["k_cache"])
    vc2 = np.empty_like(kv["v_cache"])
    kc2[perm] = kv["k_cache"]
    vc2[perm] = kv["v_cache"]
    pt = kv["page_table"]
    pt2 = np.where(pt >= 0, perm[np.maximum(pt, 0)], -1).astype(np.int32)
    out2, lse2 = orc.attention(q, kc2, vc2, pt2, qo, kvl)
    np.testing.assert_array_equal(out, out2)
    np.testing.assert_array_equal(lse, lse2)


def test_dominant_key(orc):
    d, n = 32, 40
    rng = np.random.default_rng(6)
    Kt = rng.standard_normal((1, n, d)).astype(np.float32) * 0.01
    Vt = rng.standard_normal((1, n, d)).astype(np.float32)
    q = np.ones((1, 1, d), np.float32)
    Kt[0, 17] = 10.0  # z_17 = scale * 320 ~ 56.6 above the rest
    kc, vc, pt = _cache_from_tokens(Kt, Vt, 8)
    out, _ = orc.attention(q, kc, vc, pt, [0, 1], [n])
    np.testing.assert_allclose(out[0], Vt[0, 17], atol=1e-20)


def test_selected_units_match_full(orc):
    cfg = synth.CONFIGS["tiny"]
    L = synth.kv_context_lengths(cfg)
    k = np.array([2, 8, 5, 1], np.int32)
    qo = synth.indptr_from_depths(k)
    kv = synth.make_kv(cfg, L)
    q = synth.pack_rows(kv["q_full"], qo)
    full, lf = orc.attention(q, kv["k_cache"], kv["v_cache"], kv["page_table"], qo, L + k)
    rows = np.array([0, 3, 9, 15, 15], np.int32)
    heads = np.array([0, 7, 3, 2, 5], np.int32)
    sub, ls = orc.attention(q, kv["k_cache"], kv["v_cache"], kv["page_table"], qo, L + k,
                            units=(rows, heads))
    np.testing.assert_array_equal(sub, full[rows * cfg.Hq + heads])
    np.testing.assert_array_equal(ls, lf[rows * cfg.Hq + heads])
