"""Pins of the oracle's packing and cache append: the packed batch against the budget's
own keep counts, a hand-worked example, malformed requests, and the append read back
through the page table (with every other slot unchanged), plus a round trip through the
attention oracle: appending the block and attending equals attending over a cache that
was filled with the block from the start."""
import numpy as np

import oracle
from paper_2607_25852_amd import synth


def test_pack_hand_example():
    bt = np.array([[10, 11, 12], [20, 21, 22], [30, 31, 32]], np.int32)
    qo = np.array([0, 2, 3, 6], np.int32)
    toks, pos, kvl = oracle.pack_verify(bt, [5, 0, 7], qo, 8)
    assert toks.tolist() == [10, 11, 20, 30, 31, 32, -1, -1]
    assert pos.tolist() == [5, 6, 0, 7, 8, 9, -1, -1]
    assert kvl.tolist() == [7, 1, 10]


def test_pack_follows_the_budget_and_rejects_malformed():
    rng = np.random.default_rng(0)
    R, b = 9, 6
    conf = rng.random((R, b - 1)).astype(np.float32)
    res = oracle.budget(conf, "fixed", fixed_budget=25)
    qo = res["qo_indptr"]
    bt = rng.integers(0, 1000, size=(R, b)).astype(np.int32)
    L = rng.integers(0, 300, size=R).astype(np.int32)
    toks, pos, kvl = oracle.pack_verify(bt, L, qo, 30)
    for i in range(R):
        k = res["keep"][i] + 1
        rows = np.arange(qo[i], qo[i + 1])
        assert len(rows) == k
        assert toks[rows].tolist() == bt[i, :k].tolist()
        assert pos[rows].tolist() == list(range(L[i], L[i] + k))
        assert kvl[i] == L[i] + k
    assert (toks[qo[-1]:] == -1).all()
    bad = qo.copy()
    bad[2] = bad[1]  # request 1 keeps nothing: malformed
    _, _, kvl2 = oracle.pack_verify(bt, L, bad, 30)
    assert kvl2[1] == L[1]


def test_append_read_back_and_attention_round_trip():
    cfg = synth.CONFIGS["tiny"]
    L = synth.kv_context_lengths(cfg)
    full = synth.make_kv(cfg, L)  # cache already holding L_i + b tokens per request
    qo = synth.indptr_from_depths(np.array([8, 3, 1, 6], np.int32))
    R, b, Hkv, d, P = cfg.R, cfg.b, cfg.Hkv, cfg.d, cfg.page
    # the block's keys/values as packed rows, taken from the full cache
    k_new = np.zeros((int(qo[-1]), Hkv, d), np.float32)
    v_new = np.zeros_like(k_new)
    pt = full["page_table"]
    for i in range(R):
        for j in range(int(qo[i + 1] - qo[i])):
            s = L[i] + j
            k_new[qo[i] + j] = full["k_cache"][pt[i, s // P], :, s % P]
            v_new[qo[i] + j] = full["v_cache"][pt[i, s // P], :, s % P]
    # a cache without the block: those slots hold something else
    kc0 = full["k_cache"].copy()
    vc0 = full["v_cache"].copy()
    for i in range(R):
        for j in range(b):
            s = L[i] + j
            kc0[pt[i, s // P], :, s % P] = 7.0
            vc0[pt[i, s // P], :, s % P] = -7.0
    kc, vc = oracle.append_kv(k_new, v_new, pt, qo, L, kc0, vc0, b)
    changed = np.zeros((kc.shape[0], kc.shape[2]), bool)  # (page, slot)
    for i in range(R):
        for j in range(int(qo[i + 1] - qo[i])):
            s = L[i] + j
            np.testing.assert_array_equal(kc[pt[i, s // P], :, s % P], k_new[qo[i] + j])
            np.testing.assert_array_equal(vc[pt[i, s // P], :, s % P], v_new[qo[i] + j])
            changed[pt[i, s // P], s % P] = True
    assert changed.sum() == int(qo[-1])
    for a, a0 in ((kc, kc0), (vc, vc0)):
        np.testing.assert_array_equal(a.transpose(0, 2, 1, 3)[~changed],
                                      a0.transpose(0, 2, 1, 3)[~changed])
    _, _, kvl = oracle.pack_verify(np.zeros((R, b), np.int32), L, qo, int(qo[-1]))
    q = synth.pack_rows(full["q_full"], qo)
    o1, l1 = oracle.attention(q, kc, vc, pt, qo, kvl)
    o2, l2 = oracle.attention(q, full["k_cache"], full["v_cache"], pt, qo, kvl)
    np.testing.assert_array_equal(o1, o2)
    np.testing.assert_array_equal(l1, l2)
