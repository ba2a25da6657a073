"""sv_verify_attn on the GPU against the fp64 oracle.

Gate: max-abs <= 2e-2 (bf16) / 1e-5 (fp32) plus relative RMS <= 1e-2 (bf16) /
1e-5 (fp32) and |lse difference| <= 1e-3 / 1e-5 -- at 64K-128K keys the outputs
shrink to ~1/sqrt(L), so the max-abs gate alone would pass an all-zero output.
The concurrency-64 round is compared on every (row, head) of the packing its own
budget chooses (the attention the bench times), the long-context round on every
(row, head) of eight whole requests, and every point of the concurrency sweep on the
budget's packing: every unit up to 8 requests, otherwise sampled (row, head) units
covering every request, the first and last block row and every kv-head group.
"""
import dataclasses

import numpy as np
import pytest

from gpu_util import SWEEP, bf16_bits_of, budget_packing, compare_attention, f32_of_bits, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2607_25852_amd import binding
    binding.load()
    return torch


def run_gpu_attn(torch, cfg, kv, qo, L, kv_split=0, block=None, sm_scale=0.0):
    from paper_2607_25852_amd import binding as B
    from paper_2607_25852_amd import synth
    from paper_2607_25852_amd.round import to_dev
    k = np.diff(qo)
    R = cfg.R
    q_rows = int(qo[-1])
    q = synth.pack_rows(kv["q_full"], qo)
    kv_lens = (L + k).astype(np.int32)
    blk = block or cfg.b
    d = B.attn_desc(R, q_rows, blk, cfg.Hq, cfg.Hkv, cfg.d, cfg.page, kv["page_table"].shape[1],
                    kv["num_pages"], int(kv_lens.max()), B.SV_F32 if cfg.dtype == "f32" else B.SV_BF16,
                    sm_scale=sm_scale, kv_split=kv_split)
    dt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
    out = torch.full((q_rows, cfg.Hq, cfg.d), float("nan"), dtype=dt, device="cuda")
    lse = torch.full((q_rows, cfg.Hq), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(B.attn_workspace_size(d), 256), dtype=torch.uint8, device="cuda")
    B.verify_attn(d, to_dev(q), to_dev(kv["k_cache"]), to_dev(kv["v_cache"]), to_dev(kv["page_table"]),
                  to_dev(np.ascontiguousarray(qo, np.int32)), to_dev(kv_lens), out, lse, ws)
    torch.cuda.synchronize()
    o = out.float().cpu().numpy() if cfg.dtype == "bf16" else out.cpu().numpy()
    return q, kv_lens, o.astype(np.float64), lse.cpu().numpy().astype(np.float64)


def sample_units(qo, Hq, G, n_per_req, rng):
    rows, heads = [], []
    for i in range(len(qo) - 1):
        r0, r1 = int(qo[i]), int(qo[i + 1])
        cand_rows = [r0, r1 - 1] + list(rng.integers(r0, r1, size=max(0, n_per_req - 2)))
        for j, r in enumerate(cand_rows):
            rows.append(r)
            heads.append(int((j * G + rng.integers(0, G)) % Hq) if j < Hq // G else int(rng.integers(0, Hq)))
    return np.array(rows, np.int32), np.array(heads, np.int32)


def check(orc, cfg, kv, qo, kv_lens, q, o_gpu, lse_gpu, units=None, scale=None):
    ref_o, ref_l = orc.attention(q, kv["k_cache"], kv["v_cache"], kv["page_table"], qo, kv_lens,
                                 dtype=cfg.dtype, units=units, scale=scale)
    if units is None:
        g_o = o_gpu.reshape(-1, cfg.d)
        g_l = lse_gpu.reshape(-1)
    else:
        g_o = o_gpu[units[0], units[1]]
        g_l = lse_gpu[units[0], units[1]]
    ok, stats = compare_attention(g_o, g_l, ref_o, ref_l, cfg.dtype)
    say("attn", cfg.name, stats)
    assert ok, stats
    return stats


@pytest.mark.parametrize("page,d", [(16, 64), (1, 4), (64, 100), (1, 128), (64, 256), (16, 100)])
def test_tiny_fp32_full(dev, orc, page, d):
    """fp32 path at 1e-5: head dims from 4 to 256 (100: not a multiple of 64), pages of 1 to
    64 tokens, NaN in every page and slot nobody owns, and a context of 4100 keys so that
    each of the four waves walks many 64-key tiles."""
    from paper_2607_25852_amd import synth
    cfg = dataclasses.replace(synth.CONFIGS["tiny"], name=f"tiny_f32_p{page}_d{d}", page=page, d=d,
                              kv=("list", 37, 128, 255, 4100))
    L = synth.kv_context_lengths(cfg)
    kv = synth.make_kv(cfg, L, fill_unused=np.nan)
    qo = synth.indptr_from_depths(np.array([8, 3, 1, 8]))
    say("attn tiny fp32", page, d)
    q, kvl, o, l = run_gpu_attn(dev, cfg, kv, qo, L)
    check(orc, cfg, kv, qo, kvl, q, o, l)


@pytest.mark.parametrize("page,d,k_pattern", [(16, 64, "ragged"), (64, 128, "ragged"), (16, 128, "ones"),
                                              (1, 64, "full"), (256, 128, "ragged")])
def test_tiny_bf16_full(dev, orc, page, d, k_pattern):
    from paper_2607_25852_amd import synth
    cfg = dataclasses.replace(synth.CONFIGS["tiny"], name=f"tiny_bf16_p{page}_d{d}", dtype="bf16", page=page, d=d)
    L = synth.kv_context_lengths(cfg)
    kv = synth.make_kv(cfg, L, fill_unused=np.nan)
    k = {"ragged": np.array([8, 3, 1, 6]), "ones": np.ones(4, int), "full": np.full(4, 8)}[k_pattern]
    qo = synth.indptr_from_depths(k)
    say("attn tiny bf16", page, d, k_pattern)
    q, kvl, o, l = run_gpu_attn(dev, cfg, kv, qo, L)
    check(orc, cfg, kv, qo, kvl, q, o, l)


def test_c16_b16_full(dev, orc):
    from paper_2607_25852_amd import synth
    cfg = synth.CONFIGS["c16_b16"]
    L = synth.kv_context_lengths(cfg)
    kv = synth.make_kv(cfg, L, fill_unused=np.nan)
    qo = budget_packing("c16_b16")
    say("attn c16_b16")
    q, kvl, o, l = run_gpu_attn(dev, cfg, kv, qo, L)
    rows = np.repeat(np.arange(int(qo[-1])), cfg.Hq).astype(np.int32)
    heads = np.tile(np.arange(cfg.Hq), int(qo[-1])).astype(np.int32)
    check(orc, cfg, kv, qo, kvl, q, o, l, units=(rows, heads))


def all_units(qo, Hq, rows=None):
    rows = np.arange(int(qo[-1])) if rows is None else np.asarray(rows)
    return (np.repeat(rows, Hq).astype(np.int32), np.tile(np.arange(Hq), len(rows)).astype(np.int32))


def test_c64_b16_every_unit_on_budget_packing(dev, orc):
    """The attention the bench times: the concurrency-64 round on the packing its own budget
    chooses (K = 512 of 1024 positions), every (row, head) against the oracle. The GPU
    budget's packing is checked to be that same packing first."""
    from paper_2607_25852_amd import binding as B
    from paper_2607_25852_amd import synth
    from gpu_util import conf_of
    cfg = synth.CONFIGS["c64_b16"]
    qo = budget_packing("c64_b16")
    assert int(qo[-1]) == 512
    conf = dev.from_numpy(np.ascontiguousarray(conf_of("c64_b16"))).cuda()
    bd = B.budget_desc(cfg.R, cfg.b, "cost", ratios_pm=synth.PAPER_RATIOS_PM, cost=synth.profiled_cost(cfg.R, cfg.b))
    keep = dev.empty(cfg.R, dtype=dev.int32, device="cuda")
    qo_d = dev.empty(cfg.R + 1, dtype=dev.int32, device="cuda")
    sel = dev.empty(2, dtype=dev.int32, device="cuda")
    B.alloc_budget(bd, conf, keep, qo_d, sel)
    np.testing.assert_array_equal(qo_d.cpu().numpy(), qo)
    L = synth.kv_context_lengths(cfg)
    say("attn gen c64_b16")
    kv = synth.make_kv(cfg, L)
    say("attn run c64_b16")
    q, kvl, o, l = run_gpu_attn(dev, cfg, kv, qo, L)
    check(orc, cfg, kv, qo, kvl, q, o, l, units=all_units(qo, cfg.Hq))


def test_long_c32_whole_requests(dev, orc):
    """Long context (64K-128K keys, group 16): every (row, head) of eight whole requests,
    among them the shortest and longest context, the smallest and largest block, and
    blocks of 9-10 and 11-12 rows (144..192 query rows per kv-head group)."""
    from paper_2607_25852_amd import synth
    cfg = synth.CONFIGS["long_c32"]
    L = synth.kv_context_lengths(cfg)
    qo = budget_packing("long_c32")
    k = np.diff(qo)
    pick = {int(np.argmin(L)), int(np.argmax(L)), int(np.argmin(k)), int(np.argmax(k))}
    pick |= {int(np.flatnonzero((k >= 9) & (k <= 10))[0]), int(np.flatnonzero((k >= 11) & (k <= 12))[0])}
    for i in np.random.default_rng(5).permutation(cfg.R):
        if len(pick) == 8:
            break
        pick.add(int(i))
    rows = np.concatenate([np.arange(qo[i], qo[i + 1]) for i in sorted(pick)])
    say("attn gen long_c32")
    kv = synth.make_kv(cfg, L)
    say("attn run long_c32")
    q, kvl, o, l = run_gpu_attn(dev, cfg, kv, qo, L)
    check(orc, cfg, kv, qo, kvl, q, o, l, units=all_units(qo, cfg.Hq, rows))


@pytest.mark.parametrize("name", SWEEP)
def test_sweep_on_budget_packing(dev, orc, name):
    """Every concurrency and drafter mode of the sweep (the split rule takes different
    values across them), on the packing each round's budget chooses."""
    from paper_2607_25852_amd import synth
    cfg = synth.CONFIGS[name]
    L = synth.kv_context_lengths(cfg)
    qo = budget_packing(name)
    say("attn gen", name)
    kv = synth.make_kv(cfg, L)
    say("attn run", name)
    q, kvl, o, l = run_gpu_attn(dev, cfg, kv, qo, L)
    if cfg.R <= 8:
        units = all_units(qo, cfg.Hq)
    else:
        units = sample_units(qo, cfg.Hq, cfg.Hq // cfg.Hkv, 8, np.random.default_rng(1))
    check(orc, cfg, kv, qo, kvl, q, o, l, units=units)


def test_peaky_queries_and_split_invariance(dev, orc):
    """q scaled by 4 makes outputs O(1); results must not depend on the split size."""
    from paper_2607_25852_amd import synth
    cfg = dataclasses.replace(synth.CONFIGS["c16_b16"], name="c16_peaky", R=6)
    L = synth.kv_context_lengths(synth.CONFIGS["c16_b16"])[:6]
    kv = synth.make_kv(cfg, L, q_scale=4.0, fill_unused=np.nan)
    qo = synth.indptr_from_depths(np.array([16, 1, 7, 16, 2, 11]))
    outs = []
    for split in (64, 320, 4096, 0):
        say("attn split", split)
        q, kvl, o, l = run_gpu_attn(dev, cfg, kv, qo, L, kv_split=split)
        outs.append((o, l))
    rows = np.repeat(np.arange(int(qo[-1])), cfg.Hq).astype(np.int32)
    heads = np.tile(np.arange(cfg.Hq), int(qo[-1])).astype(np.int32)
    st = check(orc, cfg, kv, qo, kvl, q, outs[0][0], outs[0][1], units=(rows, heads))
    assert st["rel_rms"] < 1e-2
    for o, l in outs[1:]:
        assert np.abs(o - outs[0][0]).max() <= 2e-2
        assert np.abs(l - outs[0][1]).max() <= 1e-3


def test_context_free_block(dev, orc):
    """L_i = 0: the block attends only to itself (row 0 sees one key)."""
    from paper_2607_25852_amd import synth
    cfg = dataclasses.replace(synth.CONFIGS["tiny"], name="nolctx", dtype="bf16", kv=("list", 0, 0, 0, 0))
    L = np.zeros(4, np.int32)
    kv = synth.make_kv(cfg, L, fill_unused=np.nan)
    qo = synth.indptr_from_depths(np.array([1, 8, 4, 2]))
    q, kvl, o, l = run_gpu_attn(dev, cfg, kv, qo, L)
    check(orc, cfg, kv, qo, kvl, q, o, l)
    # row 0 of request 0 sees exactly one key: output == its V row (rounded to bf16)
    v0 = f32_of_bits(kv["v_cache"][kv["page_table"][0, 0], 0, 0]).astype(np.float64)
    np.testing.assert_allclose(o[0, 0], v0, atol=1e-2)


def test_repeatable_bitwise(dev):
    from paper_2607_25852_amd import synth
    cfg = dataclasses.replace(synth.CONFIGS["c16_b16"], name="rep", R=4)
    L = synth.kv_context_lengths(synth.CONFIGS["c16_b16"])[:4]
    kv = synth.make_kv(cfg, L)
    qo = synth.indptr_from_depths(np.array([16, 5, 9, 1]))
    a = run_gpu_attn(dev, cfg, kv, qo, L, kv_split=256)
    b = run_gpu_attn(dev, cfg, kv, qo, L, kv_split=256)
    np.testing.assert_array_equal(a[2], b[2])
    np.testing.assert_array_equal(a[3], b[3])


def test_request_index_above_32767(dev, orc):
    """The work list encodes (request, split) in 32 bits: requests at index >= 32768
    (split partials and merge included) must come out like the others."""
    from paper_2607_25852_amd import synth
    R, tail = 32800, 40
    L = np.full(R, 5, np.int32)
    L[R - tail:] = np.random.default_rng(7).integers(100, 300, size=tail)
    cfg = dataclasses.replace(synth.CONFIGS["tiny"], name="many_reqs", R=R, b=2, dtype="bf16",
                              Hq=4, Hkv=1, d=64, page=16, kv=("list",) + tuple(int(x) for x in L))
    say("attn gen many_reqs")
    kv = synth.make_kv(cfg, L)
    qo = synth.indptr_from_depths(np.where(np.arange(R) % 2 == 0, 2, 1).astype(np.int32))
    say("attn run many_reqs")
    q, kvl, o, l = run_gpu_attn(dev, cfg, kv, qo, L, kv_split=64)
    sel = list(range(R - tail, R)) + [0, 1, 12345, 32767]
    rows = np.concatenate([np.arange(qo[i], qo[i + 1]) for i in sel]).astype(np.int32)
    rows = np.repeat(rows, cfg.Hq).astype(np.int32)
    heads = np.tile(np.arange(cfg.Hq), len(rows) // cfg.Hq).astype(np.int32)
    check(orc, cfg, kv, qo, kvl, q, o, l, units=(rows, heads))


@pytest.mark.parametrize("page,d", [(64, 128), (16, 128), (64, 64), (16, 64)])
def test_wide_group_whole_tile_waves(dev, orc, page, d):
    """More than 128 query rows per kv-head group (G = 32, block 16: up to 512 rows):
    waves own whole tiles, 256 rows per row block, partly filled blocks included."""
    from paper_2607_25852_amd import synth
    cfg = dataclasses.replace(synth.CONFIGS["tiny"], name=f"wide_p{page}_d{d}", b=16, dtype="bf16", Hq=32, Hkv=1,
                              d=d, page=page)
    L = synth.kv_context_lengths(cfg)
    kv = synth.make_kv(cfg, L, fill_unused=np.nan)
    qo = synth.indptr_from_depths(np.array([16, 3, 9, 12]))
    say("attn wide", page, d)
    q, kvl, o, l = run_gpu_attn(dev, cfg, kv, qo, L)
    check(orc, cfg, kv, qo, kvl, q, o, l)
    # the same rows through several splits agree with the single-split result
    q2, kvl2, o2, l2 = run_gpu_attn(dev, cfg, kv, qo, L, kv_split=128)
    assert np.abs(o2 - o).max() <= 2e-2 and np.abs(l2 - l).max() <= 1e-3



def test_longest_context(dev, orc):
    """A request at the longest accepted context (2^22 tokens with its block, 65536 pages of
    64): 2048 splits of 2048 tokens merged per row, next to a shorter request. The cache
    holds random bf16 values of magnitude [0.5, 1) with random signs (cheap to generate at
    this size) behind a shuffled page table."""
    from paper_2607_25852_amd import synth
    L = np.array([(1 << 22) - 4, 300001], np.int32)
    cfg = dataclasses.replace(synth.CONFIGS["tiny"], name="longest", R=2, b=4, dtype="bf16", Hq=8, Hkv=1, d=128,
                              page=64, kv=("list",) + tuple(int(x) for x in L))
    qo = synth.indptr_from_depths(np.array([4, 3], np.int32))
    say("attn gen longest")
    rng = np.random.default_rng(21)
    need = [-(-(int(L[i]) + cfg.b) // cfg.page) for i in range(cfg.R)]
    pool = sum(need)
    perm = rng.permutation(pool).astype(np.int32)
    pt = np.full((cfg.R, max(need)), -1, np.int32)
    pt[0, :need[0]] = perm[:need[0]]
    pt[1, :need[1]] = perm[need[0]:]

    def cache():
        bits = rng.integers(0, 1 << 16, size=(pool, cfg.Hkv, cfg.page, cfg.d), dtype=np.uint16)
        return (bits & np.uint16(0x807F)) | np.uint16(0x3F00)

    # queries scaled by 8: a few keys dominate each row, so a lost or misplaced split moves
    # the output and the lse by O(1)
    q32 = rng.standard_normal((cfg.R, cfg.b, cfg.Hq, cfg.d), dtype=np.float32) * np.float32(8.0)
    kv = dict(q_full=synth.bf16_bits(q32), page_table=pt, num_pages=pool, k_cache=cache(), v_cache=cache())
    say("attn run longest")
    q, kvl, o, l = run_gpu_attn(dev, cfg, kv, qo, L)
    assert int(kvl.max()) == 1 << 22
    rows = np.array([0, 0, 3, 3, 4, 4, 5, 6], np.int32)
    heads = np.array([0, 5, 2, 7, 1, 6, 3, 4], np.int32)
    check(orc, cfg, kv, qo, kvl, q, o, l, units=(rows, heads))
