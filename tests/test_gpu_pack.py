"""sv_pack_verify and sv_append_kv on the GPU against the oracle, bit for bit.

Both are integer and copy work: the packed tokens, positions and key counts, and the
whole K and V caches after the append (every byte, so a stray write anywhere fails),
must equal the oracle's. Cases cover malformed requests (k_i = 0, k_i > b, rows past
total_max), page sizes below, at and above the 64-token tile, fp32 and bf16 rows,
invalid page ids and page columns (skipped rows), and the full c64_b16 shape with
contexts up to 32768 tokens.
"""
import numpy as np
import pytest

import oracle
from gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2607_25852_amd import binding
    binding.load()
    return torch


def _qo(depths):
    qo = np.zeros(len(depths) + 1, np.int32)
    qo[1:] = np.cumsum(depths)
    return qo


def gpu_pack(torch, bt, L, qo, total_max):
    from paper_2607_25852_amd import binding as B
    from paper_2607_25852_amd.round import to_dev
    R, b = bt.shape
    toks = torch.full((total_max,), -1, dtype=torch.int32, device="cuda")
    pos = torch.full((total_max,), -1, dtype=torch.int32, device="cuda")
    kvl = torch.full((R,), -5, dtype=torch.int32, device="cuda")
    B.pack_verify(B.pack_desc(R, b, total_max), to_dev(bt), to_dev(np.asarray(L, np.int32)),
                  to_dev(np.asarray(qo, np.int32)), toks, pos, kvl)
    torch.cuda.synchronize()
    return toks.cpu().numpy(), pos.cpu().numpy(), kvl.cpu().numpy()


@pytest.mark.parametrize("R,b,seed", [(1, 1, 0), (7, 5, 1), (64, 16, 2), (1000, 16, 3), (70000, 4, 4)])
def test_pack_bit_exact(dev, R, b, seed):
    say(f"pack R={R} b={b} seed={seed}")
    rng = np.random.default_rng(seed)
    k = rng.integers(1, b + 1, size=R).astype(np.int32)
    if R > 2:
        k[rng.integers(0, R)] = 0          # malformed: keeps nothing
        k[rng.integers(0, R)] = b + 1      # malformed: more than the block
    qo = _qo(k)
    total_max = int(qo[-1]) - (2 if R > 2 else 0)  # the last request's rows overrun
    total_max = max(total_max, 1)
    bt = rng.integers(0, 1 << 30, size=(R, b)).astype(np.int32)
    L = rng.integers(0, 1 << 22, size=R).astype(np.int32)
    got = gpu_pack(dev, bt, L, qo, total_max)
    want = oracle.pack_verify(bt, L, qo, total_max)
    for g, w, name in zip(got, want, ("tokens", "positions", "kv_lens")):
        np.testing.assert_array_equal(g, w, err_msg=name)


def _cache(rng, shape, dtype):
    if dtype == "f32":
        return rng.standard_normal(shape, dtype=np.float32)
    return rng.integers(0, 1 << 16, size=shape).astype(np.uint16)


def gpu_append(torch, k_new, v_new, pt, qo, L, kc, vc, block, dtype):
    from paper_2607_25852_amd import binding as B
    from paper_2607_25852_amd.round import to_dev
    R, maxp = pt.shape
    num_pages, Hkv, P, d = kc.shape
    desc = B.append_desc(R, k_new.shape[0], block, Hkv, d, P, maxp, num_pages, B.SV_F32 if dtype == "f32" else B.SV_BF16)
    kc_d, vc_d = to_dev(kc), to_dev(vc)
    B.append_kv(desc, to_dev(k_new), to_dev(v_new), to_dev(pt), to_dev(np.asarray(qo, np.int32)),
                to_dev(np.asarray(L, np.int32)), kc_d, vc_d)
    torch.cuda.synchronize()
    out = []
    for t in (kc_d, vc_d):
        a = t.cpu()
        out.append(a.view(torch.int16).numpy().view(np.uint16) if dtype == "bf16" else a.numpy())
    return out


def _append_case(rng, R, b, Hkv, d, P, dtype, max_ctx, bad=True, slack=1.3):
    k = rng.integers(1, b + 1, size=R).astype(np.int32)
    L = rng.integers(0, max_ctx + 1, size=R).astype(np.int32)
    need = [(-(-(int(L[i]) + b) // P)) for i in range(R)]
    maxp = max(need)
    pool = int(np.ceil(sum(-(-b // P) + 1 for _ in range(R)) * slack)) + 2
    # only the page columns the block can touch are mapped; the rest are -1
    pt = np.full((R, maxp), -1, np.int32)
    perm = rng.permutation(pool).astype(np.int32)
    cur = 0
    for i in range(R):
        for col in range(int(L[i]) // P, need[i]):
            pt[i, col] = perm[cur]
            cur += 1
    assert cur <= pool
    if bad and R > 3:
        i = int(rng.integers(0, R))
        pt[i, int(L[i]) // P] = pool + 3          # page id past the pool: skipped
        k[int(rng.integers(0, R))] = 0            # request keeps nothing
        j = int(rng.integers(0, R))
        L[j] = maxp * P - 1                       # block runs past the last page column
        k[j] = min(b, 2) if b >= 2 else 1
        pt[j, maxp - 1] = perm[-1]
    qo = _qo(k)
    total = int(qo[-1]) + 3
    k_new = _cache(rng, (total, Hkv, d), dtype)
    v_new = _cache(rng, (total, Hkv, d), dtype)
    kc = _cache(rng, (pool, Hkv, P, d), dtype)
    vc = _cache(rng, (pool, Hkv, P, d), dtype)
    return k_new, v_new, pt, qo, L, kc, vc


@pytest.mark.parametrize("R,b,Hkv,d,P,dtype,seed", [
    (1, 1, 1, 4, 1, "f32", 0),
    (5, 8, 2, 64, 16, "f32", 1),
    (9, 16, 8, 128, 64, "bf16", 2),
    (33, 5, 1, 64, 256, "bf16", 3),
    (17, 16, 4, 128, 1, "bf16", 4),
    (12, 3, 3, 20, 8, "f32", 5),
])
def test_append_bit_exact(dev, R, b, Hkv, d, P, dtype, seed):
    say(f"append R={R} b={b} Hkv={Hkv} d={d} P={P} {dtype} seed={seed}")
    rng = np.random.default_rng(100 + seed)
    k_new, v_new, pt, qo, L, kc, vc = _append_case(rng, R, b, Hkv, d, P, dtype, 3000)
    gk, gv = gpu_append(dev, k_new, v_new, pt, qo, L, kc, vc, b, dtype)
    wk, wv = oracle.append_kv(k_new, v_new, pt, qo, L, kc, vc, b)
    np.testing.assert_array_equal(gk, wk)
    np.testing.assert_array_equal(gv, wv)
    assert (gk != kc).any() or int(qo[-1]) == 0  # something was written


@pytest.mark.parametrize("seed", range(24))
def test_append_random_shapes(dev, seed):
    """Random shapes (requests, block, kv-heads, row lengths of 16-byte multiples up to
    256 elements, pages of 1-512 tokens, bf16 and fp32), each with the malformed requests
    of the fixed cases: the whole caches equal the oracle's, bit for bit."""
    rng = np.random.default_rng(7000 + seed)
    dtype = "f32" if seed % 3 == 0 else "bf16"
    unit = 4 if dtype == "f32" else 8
    R = int(rng.integers(1, 48))
    b = int(rng.integers(1, 17))
    Hkv = int(rng.integers(1, 9))
    d = unit * int(rng.integers(1, 256 // unit + 1))
    P = 1 << int(rng.integers(0, 10))
    say(f"append random seed={seed} R={R} b={b} Hkv={Hkv} d={d} P={P} {dtype}")
    k_new, v_new, pt, qo, L, kc, vc = _append_case(rng, R, b, Hkv, d, P, dtype, 2000)
    gk, gv = gpu_append(dev, k_new, v_new, pt, qo, L, kc, vc, b, dtype)
    wk, wv = oracle.append_kv(k_new, v_new, pt, qo, L, kc, vc, b)
    np.testing.assert_array_equal(gk, wk)
    np.testing.assert_array_equal(gv, wv)


def test_append_full_c64_b16_shape(dev):
    """The c64_b16 launch shape (64 requests, block 16, 8 kv-heads, d 128, 64-token
    pages, bf16) with contexts up to 32768 tokens."""
    say("append c64_b16 shape")
    rng = np.random.default_rng(7)
    k_new, v_new, pt, qo, L, kc, vc = _append_case(rng, 64, 16, 8, 128, 64, "bf16", 32768, bad=False)
    gk, gv = gpu_append(dev, k_new, v_new, pt, qo, L, kc, vc, 16, "bf16")
    wk, wv = oracle.append_kv(k_new, v_new, pt, qo, L, kc, vc, 16)
    np.testing.assert_array_equal(gk, wk)
    np.testing.assert_array_equal(gv, wv)


def test_pack_append_then_attend(dev):
    """Packing, appending the block's keys and values into slots that held NaN, then
    sv_verify_attn, equals the oracle's attention over the cache that held the block
    from the start (the append puts every key at the position attention reads)."""
    from paper_2607_25852_amd import binding as B
    from paper_2607_25852_amd import synth
    from paper_2607_25852_amd.round import to_dev
    from gpu_util import compare_attention
    torch = dev
    cfg = synth.CONFIGS["c16_b16"]
    say("pack+append+attend c16_b16")
    L = synth.kv_context_lengths(cfg)
    full = synth.make_kv(cfg, L)
    pt = full["page_table"]
    P, b, R = cfg.page, cfg.b, cfg.R
    qo = synth.indptr_from_depths(synth.given_depths(cfg))
    rows = int(qo[-1])
    k_new = np.zeros((rows, cfg.Hkv, cfg.d), np.uint16)
    v_new = np.zeros_like(k_new)
    kc0, vc0 = full["k_cache"].copy(), full["v_cache"].copy()
    nan = synth.bf16_bits(np.array([np.nan], np.float32))[0]
    for i in range(R):
        for j in range(b):
            s = int(L[i]) + j
            if j < qo[i + 1] - qo[i]:
                k_new[qo[i] + j] = full["k_cache"][pt[i, s // P], :, s % P]
                v_new[qo[i] + j] = full["v_cache"][pt[i, s // P], :, s % P]
            kc0[pt[i, s // P], :, s % P] = nan
            vc0[pt[i, s // P], :, s % P] = nan
    toks, pos, kvl = gpu_pack(torch, np.zeros((R, b), np.int32), L, qo, rows)
    assert (pos == oracle.pack_verify(np.zeros((R, b), np.int32), L, qo, rows)[1]).all()
    desc = B.append_desc(R, rows, b, cfg.Hkv, cfg.d, P, pt.shape[1], full["num_pages"], B.SV_BF16)
    kc_d, vc_d = to_dev(kc0), to_dev(vc0)
    pt_d, qo_d = to_dev(pt), to_dev(np.asarray(qo, np.int32))
    B.append_kv(desc, to_dev(k_new), to_dev(v_new), pt_d, qo_d, to_dev(np.asarray(L, np.int32)), kc_d, vc_d)
    q = synth.pack_rows(full["q_full"], qo)
    ad = B.attn_desc(R, rows, b, cfg.Hq, cfg.Hkv, cfg.d, P, pt.shape[1], full["num_pages"], int(kvl.max()), B.SV_BF16)
    out = torch.empty((rows, cfg.Hq, cfg.d), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((rows, cfg.Hq), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(B.attn_workspace_size(ad), 256), dtype=torch.uint8, device="cuda")
    B.verify_attn(ad, to_dev(q), kc_d, vc_d, pt_d, qo_d, to_dev(kvl), out, lse, ws)
    torch.cuda.synchronize()
    o_ref, lse_ref = oracle.attention(q, full["k_cache"], full["v_cache"], pt, qo, kvl, dtype="bf16")
    ok, stats = compare_attention(out.float().cpu().numpy().reshape(-1, cfg.d),
                                  lse.cpu().numpy().reshape(-1), o_ref, lse_ref, "bf16")
    say("pack+append+attend", stats)
    assert ok, stats
