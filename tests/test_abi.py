"""C-ABI checks that need no GPU: the library loads, exports every symbol the header
declares, and rejects invalid calls on the host before anything is enqueued.
NULL data pointers are used throughout, so no call here can reach a kernel launch
even if a check were missing (the pointer checks would stop it first)."""
import ctypes
import os
import re

import pytest

from paper_2607_25852_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "specverify.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        from paper_2607_25852_amd import build
        build.build()
    return B.load()


def test_header_declarations_are_exported(lib):
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    declared = set(re.findall(r"\b(sv_[a-z_]+)\s*\(", text))
    assert declared == set(B.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name


def test_version_and_status_strings(lib):
    assert lib.sv_abi_version() == 1
    assert B.status_string(0) == "SV_OK"
    assert B.status_string(3) == "SV_ERR_WORKSPACE"
    assert B.status_string(99) == "SV_UNKNOWN_STATUS"


def _budget(lib, d, conf=None):
    return lib.sv_alloc_budget(ctypes.byref(d), conf, None, None, None, None, None, None)


@pytest.mark.parametrize("kw,status,msg", [
    (dict(R=0, b=4, mode="fixed", fixed_budget=1), 1, "num_reqs"),
    (dict(R=4097, b=1, mode="fixed", fixed_budget=4097), 1, "num_reqs"),
    (dict(R=4, b=17, mode="fixed", fixed_budget=4), 1, "block"),
    (dict(R=1024, b=16, mode="fixed", fixed_budget=1024), 2, "above 8192"),
])
def test_budget_descriptor_checks(lib, kw, status, msg):
    d = B.budget_desc(**kw)
    assert _budget(lib, d) == status
    assert msg in B.last_error()


def test_budget_argument_checks(lib):
    fake = ctypes.c_void_p(16)
    d = B.budget_desc(4, 8, "fixed", fixed_budget=3)
    # NULL outputs are rejected first
    assert _budget(lib, d) == 1 and "must not be NULL" in B.last_error()
    def call(d):
        return lib.sv_alloc_budget(ctypes.byref(d), None, fake, fake, fake, None, None, None)
    assert call(d) == 1 and "conf" in B.last_error()  # conf NULL with b > 1
    def call2(d):
        return lib.sv_alloc_budget(ctypes.byref(d), None, None, None, None, None, None, None)
    d = B.budget_desc(4, 8, "fixed", fixed_budget=33)
    assert call2(d) == 1
    d = B.budget_desc(4, 8, "cost", ratios_pm=(500, 250), cost=(1, 1))
    assert call2(d) == 1
    d = B.budget_desc(4, 8, "cost", ratios_pm=(250, 500), cost=(1, 0))
    assert call2(d) == 1


def _attn(lib, d, ws_bytes=0):
    return lib.sv_verify_attn(ctypes.byref(d), None, None, None, None, None, None, None, None, None, ws_bytes,
                              None)


@pytest.mark.parametrize("kw,status,msg", [
    (dict(Hq=8, Hkv=3), 1, "multiple"),
    (dict(page_size=48), 1, "power of two"),
    (dict(block=17), 1, "block"),
    (dict(d=96), 2, "head_dim"),
    (dict(Hq=128, Hkv=1), 2, "1024"),  # G = 128, 128 * 16 rows
    (dict(kv_split=100), 1, "kv_split"),
    (dict(max_pages_per_req=2), 1, "max_pages_per_req*page_size"),
    (dict(dtype=7), 1, "dtype"),
    (dict(total_q_max=65), 1, "num_reqs*block"),  # more rows than R*block
    # total_q_max * Hq would wrap in 32 bits (the fp32 path's grid of (row, head) units)
    (dict(R=65535, block=16, total_q_max=65535 * 16, Hq=4096, Hkv=4096, d=64, dtype=B.SV_F32), 2, "2^31"),
])
def test_attn_descriptor_checks(lib, kw, status, msg):
    base = dict(R=4, total_q_max=64, block=16, Hq=32, Hkv=8, d=128, page_size=64, max_pages_per_req=130,
                num_pages=1000, max_kv_len=8200, dtype=B.SV_BF16, kv_split=0)
    base.update(kw)
    d = B.attn_desc(**base)
    assert _attn(lib, d) == status
    assert msg in B.last_error()
    assert lib.sv_verify_attn_workspace_size(ctypes.byref(d)) == 0


def test_attn_workspace_size_and_null_pointers(lib):
    d = B.attn_desc(64, 1024, 16, 64, 8, 128, 64, 520, 40000, 33000, B.SV_BF16)
    n = lib.sv_verify_attn_workspace_size(ctypes.byref(d))
    assert n > 0 and n % 4 == 0
    assert _attn(lib, d) == 1 and "NULL" in B.last_error()


def _accept(lib, d, ws=None, ws_bytes=0):
    return lib.sv_spec_accept(ctypes.byref(d), None, None, None, None, None, None, None, None, None, ws, ws_bytes,
                              None)


@pytest.mark.parametrize("kw,status,msg", [
    (dict(R=0), 1, "num_reqs"),
    (dict(b=0), 1, "block"),
    (dict(V=(1 << 22) + 1), 1, "vocab"),
    (dict(kind=B.SV_PROBS, dtype=B.SV_BF16), 2, "fp32"),
    (dict(temperature=-1.0), 1, "temperature"),
    (dict(temperature=float("inf")), 1, "temperature"),
    (dict(temperature=float("nan")), 1, "temperature"),
    (dict(kind=5), 1, "kind"),
])
def test_accept_descriptor_checks(lib, kw, status, msg):
    base = dict(R=8, b=16, V=32768, kind=B.SV_LOGITS, dtype=B.SV_BF16, temperature=1.0)
    base.update(kw)
    d = B.accept_desc(**base)
    assert _accept(lib, d) == status
    assert msg in B.last_error()


def test_accept_workspace_checks(lib):
    d = B.accept_desc(8, 16, 32768, B.SV_LOGITS, B.SV_BF16)
    need = lib.sv_spec_accept_workspace_size(ctypes.byref(d))
    assert need > 0
    assert _accept(lib, d) == 1 and "NULL" in B.last_error()


def test_accept_noalloc_host_checks(lib):
    """The no-allocation variant rejects on the host, before any HIP call: a shape whose
    workspace exceeds the fixed 16 MiB scratch, then NULL pointers."""
    big = B.accept_desc(4096, 16, 131072, B.SV_LOGITS, B.SV_BF16)
    assert lib.sv_spec_accept_workspace_size(ctypes.byref(big)) > 16 << 20
    st = lib.sv_spec_accept_noalloc(ctypes.byref(big), None, None, None, None, None, None, None, None, None, None)
    assert st == B.SV_ERR_UNSUPPORTED and "16777216" in B.last_error()
    small = B.accept_desc(64, 16, 131072, B.SV_LOGITS, B.SV_BF16)
    assert lib.sv_spec_accept_workspace_size(ctypes.byref(small)) <= 16 << 20
    st = lib.sv_spec_accept_noalloc(ctypes.byref(small), None, None, None, None, None, None, None, None, None, None)
    assert st == B.SV_ERR_INVALID_ARG and "NULL" in B.last_error()
    bad = B.accept_desc(0, 16, 131072, B.SV_LOGITS, B.SV_BF16)
    st = lib.sv_spec_accept_noalloc(ctypes.byref(bad), None, None, None, None, None, None, None, None, None, None)
    assert st == B.SV_ERR_INVALID_ARG and "num_reqs" in B.last_error()


def test_error_is_thread_local(lib):
    import threading
    d = B.accept_desc(0, 16, 100, B.SV_LOGITS, B.SV_F32)
    assert _accept(lib, d) == 1
    seen = []

    def other():
        seen.append(B.last_error())

    t = threading.Thread(target=other)
    t.start()
    t.join()
    assert seen == [""] and "num_reqs" in B.last_error()


def test_injected_launch_failure_enqueues_nothing(lib, monkeypatch):
    """SV_FAULT_INJECT=launch: a valid call reports SV_ERR_HIP from the host without
    launching (the fake pointers below are never dereferenced)."""
    monkeypatch.setenv("SV_FAULT_INJECT", "launch")
    fake = ctypes.c_void_p(256)
    d = B.budget_desc(4, 8, "fixed", fixed_budget=32)
    st = lib.sv_alloc_budget(ctypes.byref(d), fake, fake, fake, fake, None, None, None)
    assert st == B.SV_ERR_HIP and "injected" in B.last_error()
    d = B.accept_desc(4, 8, 1024, B.SV_LOGITS, B.SV_F32)
    need = lib.sv_spec_accept_workspace_size(ctypes.byref(d))
    st = lib.sv_spec_accept(ctypes.byref(d), fake, fake, fake, fake, fake, fake, fake, fake, None, fake, need, None)
    assert st == B.SV_ERR_HIP
    # too-small workspace is reported before the injected failure
    st = lib.sv_spec_accept(ctypes.byref(d), fake, fake, fake, fake, fake, fake, fake, fake, None, fake, need - 1,
                            None)
    assert st == B.SV_ERR_WORKSPACE


def test_misaligned_pointers_are_rejected(lib):
    """Checked on the host before any launch (the fake addresses are never touched)."""
    ok16, odd = ctypes.c_void_p(4096), ctypes.c_void_p(4096 + 2)
    d = B.budget_desc(4, 8, "fixed", fixed_budget=32)
    st = lib.sv_alloc_budget(ctypes.byref(d), odd, ok16, ok16, ok16, None, None, None)
    assert st == B.SV_ERR_INVALID_ARG and "aligned" in B.last_error()
    d = B.attn_desc(4, 64, 16, 32, 8, 128, 64, 130, 1000, 8200, B.SV_BF16)
    need = lib.sv_verify_attn_workspace_size(ctypes.byref(d))
    args = [ok16] * 7
    for bad in range(7):
        a = list(args)
        a[bad] = ctypes.c_void_p(4096 + (8 if bad in (0, 1, 2, 6) else 2))
        st = lib.sv_verify_attn(ctypes.byref(d), *a, ok16, ok16, need, None)
        assert st == B.SV_ERR_INVALID_ARG and "aligned" in B.last_error(), bad
    d = B.accept_desc(4, 8, 1024, B.SV_LOGITS, B.SV_BF16)
    need = lib.sv_spec_accept_workspace_size(ctypes.byref(d))
    st = lib.sv_spec_accept(ctypes.byref(d), ctypes.c_void_p(4096 + 8), ok16, ok16, ok16, ok16, ok16, ok16, ok16,
                            None, ok16, need, None)
    assert st == B.SV_ERR_INVALID_ARG and "aligned" in B.last_error()


@pytest.mark.parametrize("kw,status,msg", [
    (dict(R=0), 1, "num_reqs"),
    (dict(drafts=0), 1, "drafts"),
    (dict(V=0), 1, "vocab"),
    (dict(V=(1 << 22) + 1), 1, "vocab"),
    (dict(dtype=7), 1, "dtype"),
    (dict(temperature=0.0), 1, "temperature"),
    (dict(temperature=float("nan")), 1, "temperature"),
    (dict(temperature=float("inf")), 1, "temperature"),
])
def test_draft_stats_descriptor_checks(lib, kw, status, msg):
    base = dict(R=8, drafts=15, V=32768, dtype=B.SV_BF16, temperature=1.0)
    base.update(kw)
    d = B.draft_stats_desc(base["R"], base["drafts"], base["V"], base["dtype"], base["temperature"])
    assert lib.sv_draft_stats_workspace_size(ctypes.byref(d)) == 0
    assert lib.sv_draft_stats(ctypes.byref(d), None, None, None, None, 0, None) == status
    assert msg in B.last_error()


def test_draft_stats_pointer_workspace_and_fault_checks(lib, monkeypatch):
    """NULL, misaligned and short-workspace calls are rejected on the host; with
    SV_FAULT_INJECT=launch a valid call reports SV_ERR_HIP without launching (the fake
    addresses are never touched)."""
    ok16, odd = ctypes.c_void_p(4096), ctypes.c_void_p(4096 + 4)
    d = B.draft_stats_desc(4, 7, 1000, B.SV_F32, 0.7)
    need = lib.sv_draft_stats_workspace_size(ctypes.byref(d))
    assert need == 4 * 7 * 1 * 8  # one 16 KB chunk of fp32 logits per row, a float2 each
    assert lib.sv_draft_stats(ctypes.byref(d), None, ok16, None, ok16, need, None) == 1
    assert "NULL" in B.last_error()
    assert lib.sv_draft_stats(ctypes.byref(d), ok16, odd, None, ok16, need, None) == 1
    assert "aligned" in B.last_error()
    assert lib.sv_draft_stats(ctypes.byref(d), ok16, ok16, None, ok16, need - 1, None) == B.SV_ERR_WORKSPACE
    monkeypatch.setenv("SV_FAULT_INJECT", "launch")
    assert lib.sv_draft_stats(ctypes.byref(d), ok16, ok16, ok16, ok16, need, None) == B.SV_ERR_HIP


def test_accept_stats_checks(lib, monkeypatch):
    """sv_spec_accept_stats: logits mode with T > 0 only, draft_stats required when b > 1,
    8-byte aligned; otherwise the checks of sv_spec_accept."""
    ok16 = ctypes.c_void_p(4096)
    for kind, T in ((B.SV_PROBS, 1.0), (B.SV_LOGITS, 0.0)):
        d = B.accept_desc(4, 8, 1024, kind, B.SV_F32, T)
        st = lib.sv_spec_accept_stats(ctypes.byref(d), ok16, ok16, ok16, ok16, ok16, ok16, ok16, ok16, ok16, None,
                                      ok16, 1 << 20, None)
        assert st == B.SV_ERR_INVALID_ARG and "rejection sampling" in B.last_error()
    d = B.accept_desc(4, 8, 1024, B.SV_LOGITS, B.SV_F32)
    need = lib.sv_spec_accept_workspace_size(ctypes.byref(d))
    st = lib.sv_spec_accept_stats(ctypes.byref(d), ok16, ok16, None, ok16, ok16, ok16, ok16, ok16, ok16, None, ok16,
                                  need, None)
    assert st == B.SV_ERR_INVALID_ARG and "draft_stats" in B.last_error()
    st = lib.sv_spec_accept_stats(ctypes.byref(d), ok16, ok16, ctypes.c_void_p(4096 + 4), ok16, ok16, ok16, ok16,
                                  ok16, ok16, None, ok16, need, None)
    assert st == B.SV_ERR_INVALID_ARG and "aligned" in B.last_error()
    monkeypatch.setenv("SV_FAULT_INJECT", "launch")
    st = lib.sv_spec_accept_stats(ctypes.byref(d), ok16, ok16, ok16, ok16, ok16, ok16, ok16, ok16, ok16, None, ok16,
                                  need, None)
    assert st == B.SV_ERR_HIP and "sv_spec_accept_stats" in B.last_error()


def test_probe_header_declarations_are_exported():
    """The measurement probe's header and library agree (libsvprobe.so, built with the
    main library); an invalid call is refused on the host."""
    from paper_2607_25852_amd import build
    if not os.path.exists(build.PROBE_LIB):
        build.build()
    text = open(os.path.join(ROOT, "include", "svprobe.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    declared = set(re.findall(r"\b(svprobe_[a-z_]+)\s*\(", text))
    assert declared == {"svprobe_stream_read"}
    lib = ctypes.CDLL(build.PROBE_LIB)
    lib.svprobe_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p]
    lib.svprobe_stream_read.restype = ctypes.c_int32
    assert lib.svprobe_stream_read(None, 32768, None, None) == -1
    assert lib.svprobe_stream_read(ctypes.c_void_p(4096), 1000, ctypes.c_void_p(4096), None) == -1
    assert lib.svprobe_stream_read(ctypes.c_void_p(4100), 32768, ctypes.c_void_p(4096), None) == -1



def test_prepare_round_and_attention_plan_checks(lib, monkeypatch):
    """sv_prepare_round, sv_verify_attn_plan and sv_verify_attn_run reject bad calls on the
    host (fake pointers never dereferenced; SV_FAULT_INJECT stops valid calls before any
    launch)."""
    fake = ctypes.c_void_p(256)
    bd = B.budget_desc(4, 8, "fixed", fixed_budget=32)
    pd = B.pack_desc(4, 8, 32)
    ad = B.attn_desc(4, 32, 8, 32, 8, 128, 64, 130, 1000, 8200, B.SV_BF16)
    need = lib.sv_verify_attn_workspace_size(ctypes.byref(ad))

    def prep(bdesc, pdesc, adesc, ws_bytes, ptr=fake):
        return lib.sv_prepare_round(ctypes.byref(bdesc), fake, fake, fake, fake, None, None, ctypes.byref(pdesc),
                                    ptr, fake, fake, fake, fake, None if adesc is None else ctypes.byref(adesc),
                                    fake, ws_bytes, None)
    # the packing and the attention descriptors must agree with the budget's
    assert prep(bd, B.pack_desc(5, 8, 32), None, 0) == B.SV_ERR_INVALID_ARG and "packing" in B.last_error()
    assert prep(bd, B.pack_desc(4, 9, 36), None, 0) == B.SV_ERR_INVALID_ARG and "packing" in B.last_error()
    bad_a = B.attn_desc(5, 32, 8, 32, 8, 128, 64, 130, 1000, 8200, B.SV_BF16)
    assert prep(bd, pd, bad_a, need) == B.SV_ERR_INVALID_ARG and "attention" in B.last_error()
    assert prep(bd, pd, ad, need - 1) == B.SV_ERR_WORKSPACE
    assert prep(bd, pd, ad, need, ptr=None) == B.SV_ERR_INVALID_ARG and "NULL" in B.last_error()
    assert prep(B.budget_desc(4, 8, "fixed", fixed_budget=33), pd, None, 0) == B.SV_ERR_INVALID_ARG
    # plan and run: the attention descriptor's checks, then pointers and workspace
    assert lib.sv_verify_attn_plan(ctypes.byref(B.attn_desc(4, 32, 8, 32, 3, 128, 64, 130, 1000, 8200,
                                                            B.SV_BF16)), fake, fake, fake, need,
                                   None) == B.SV_ERR_INVALID_ARG
    assert lib.sv_verify_attn_plan(ctypes.byref(ad), None, fake, fake, need, None) == B.SV_ERR_INVALID_ARG
    assert lib.sv_verify_attn_plan(ctypes.byref(ad), fake, fake, fake, need - 1, None) == B.SV_ERR_WORKSPACE
    assert lib.sv_verify_attn_run(ctypes.byref(ad), None, None, None, None, None, None, None, None, fake, need,
                                  None) == B.SV_ERR_INVALID_ARG
    assert lib.sv_verify_attn_run(ctypes.byref(ad), fake, fake, fake, fake, fake, fake, fake, None, fake, need - 1,
                                  None) == B.SV_ERR_WORKSPACE
    monkeypatch.setenv("SV_FAULT_INJECT", "launch")
    assert prep(bd, pd, ad, need) == B.SV_ERR_HIP and "sv_prepare_round" in B.last_error()
    assert lib.sv_verify_attn_plan(ctypes.byref(ad), fake, fake, fake, need, None) == B.SV_ERR_HIP
    assert lib.sv_verify_attn_run(ctypes.byref(ad), fake, fake, fake, fake, fake, fake, fake, None, fake, need,
                                  None) == B.SV_ERR_HIP
