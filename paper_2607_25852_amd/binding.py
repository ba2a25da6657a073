"""ctypes binding of libspecverify (include/specverify.h).

Argument marshalling only: torch tensors are passed as device pointers together
with the current HIP stream; every step of the round runs in the library's HIP
kernels. Loading fails loudly when the library has not been built -- there is
no fallback of any kind.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libspecverify.so")

SV_OK, SV_ERR_INVALID_ARG, SV_ERR_UNSUPPORTED, SV_ERR_WORKSPACE, SV_ERR_HIP = range(5)
SV_F32, SV_BF16 = 0, 1
SV_LOGITS, SV_PROBS = 0, 1
SV_BUDGET_FIXED, SV_BUDGET_COST = 0, 1
SV_MAX_RATIOS = 8

# every symbol the header declares (checked by the ABI test)
EXPORTED = ("sv_alloc_budget", "sv_pack_verify", "sv_append_kv", "sv_verify_attn", "sv_verify_attn_workspace_size",
            "sv_verify_attn_plan", "sv_verify_attn_run", "sv_prepare_round",
            "sv_spec_accept", "sv_spec_accept_workspace_size", "sv_spec_accept_noalloc", "sv_spec_accept_debug",
            "sv_spec_accept_stats",
            "sv_draft_stats",
            "sv_draft_stats_workspace_size", "sv_status_string", "sv_last_error", "sv_abi_version")


class BudgetDesc(ctypes.Structure):
    _fields_ = [("num_reqs", ctypes.c_int32), ("block", ctypes.c_int32), ("mode", ctypes.c_int32),
                ("fixed_budget", ctypes.c_int32), ("num_ratios", ctypes.c_int32),
                ("ratio_permille", ctypes.c_int32 * SV_MAX_RATIOS),
                ("cost", ctypes.c_uint32 * SV_MAX_RATIOS)]


class AttnDesc(ctypes.Structure):
    _fields_ = [("num_reqs", ctypes.c_int32), ("total_q_max", ctypes.c_int32), ("block", ctypes.c_int32),
                ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("max_pages_per_req", ctypes.c_int32), ("num_pages", ctypes.c_int32),
                ("max_kv_len", ctypes.c_int32), ("dtype", ctypes.c_int32), ("sm_scale", ctypes.c_float),
                ("kv_split", ctypes.c_int32)]


class AcceptDesc(ctypes.Structure):
    _fields_ = [("num_reqs", ctypes.c_int32), ("block", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("kind", ctypes.c_int32), ("dtype", ctypes.c_int32), ("temperature", ctypes.c_float)]


class DraftStatsDesc(ctypes.Structure):
    _fields_ = [("num_reqs", ctypes.c_int32), ("drafts", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("temperature", ctypes.c_float)]


class PackDesc(ctypes.Structure):
    _fields_ = [("num_reqs", ctypes.c_int32), ("block", ctypes.c_int32), ("total_max", ctypes.c_int32)]


class AppendDesc(ctypes.Structure):
    _fields_ = [("num_reqs", ctypes.c_int32), ("total_max", ctypes.c_int32), ("block", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("max_pages_per_req", ctypes.c_int32), ("num_pages", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class SpecVerifyError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{status_string(status)}: {msg}")
        self.status = status


_lib = None


def load() -> ctypes.CDLL:
    """Load libspecverify.so (raises if it was not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2607_25852_amd.build.build() "
                           "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    i32 = ctypes.c_int32
    lib.sv_alloc_budget.argtypes = [ctypes.POINTER(BudgetDesc), P, P, P, P, P, P, P]
    lib.sv_alloc_budget.restype = i32
    lib.sv_verify_attn.argtypes = [ctypes.POINTER(AttnDesc), P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P]
    lib.sv_verify_attn.restype = i32
    lib.sv_verify_attn_run.argtypes = [ctypes.POINTER(AttnDesc), P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P]
    lib.sv_verify_attn_run.restype = i32
    lib.sv_verify_attn_plan.argtypes = [ctypes.POINTER(AttnDesc), P, P, P, ctypes.c_size_t, P]
    lib.sv_verify_attn_plan.restype = i32
    lib.sv_prepare_round.argtypes = [ctypes.POINTER(BudgetDesc), P, P, P, P, P, P, ctypes.POINTER(PackDesc), P, P, P,
                                     P, P, ctypes.POINTER(AttnDesc), P, ctypes.c_size_t, P]
    lib.sv_prepare_round.restype = i32
    lib.sv_verify_attn_workspace_size.argtypes = [ctypes.POINTER(AttnDesc)]
    lib.sv_verify_attn_workspace_size.restype = ctypes.c_size_t
    lib.sv_spec_accept.argtypes = [ctypes.POINTER(AcceptDesc), P, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P]
    lib.sv_spec_accept.restype = i32
    lib.sv_spec_accept_workspace_size.argtypes = [ctypes.POINTER(AcceptDesc)]
    lib.sv_spec_accept_workspace_size.restype = ctypes.c_size_t
    lib.sv_spec_accept_noalloc.argtypes = [ctypes.POINTER(AcceptDesc), P, P, P, P, P, P, P, P, P, P]
    lib.sv_spec_accept_noalloc.restype = i32
    lib.sv_spec_accept_debug.argtypes = [ctypes.POINTER(AcceptDesc), P, P, P, P, P, P, P, P, P, P, P, P,
                                         ctypes.c_size_t, P]
    lib.sv_spec_accept_debug.restype = i32
    lib.sv_spec_accept_stats.argtypes = [ctypes.POINTER(AcceptDesc), P, P, P, P, P, P, P, P, P, P, P,
                                         ctypes.c_size_t, P]
    lib.sv_spec_accept_stats.restype = i32
    lib.sv_draft_stats.argtypes = [ctypes.POINTER(DraftStatsDesc), P, P, P, P, ctypes.c_size_t, P]
    lib.sv_draft_stats.restype = i32
    lib.sv_draft_stats_workspace_size.argtypes = [ctypes.POINTER(DraftStatsDesc)]
    lib.sv_draft_stats_workspace_size.restype = ctypes.c_size_t
    lib.sv_pack_verify.argtypes = [ctypes.POINTER(PackDesc), P, P, P, P, P, P, P]
    lib.sv_pack_verify.restype = i32
    lib.sv_append_kv.argtypes = [ctypes.POINTER(AppendDesc), P, P, P, P, P, P, P, P]
    lib.sv_append_kv.restype = i32
    lib.sv_status_string.argtypes = [i32]
    lib.sv_status_string.restype = ctypes.c_char_p
    lib.sv_last_error.argtypes = []
    lib.sv_last_error.restype = ctypes.c_char_p
    lib.sv_abi_version.argtypes = []
    lib.sv_abi_version.restype = i32
    _lib = lib
    return lib


def status_string(st: int) -> str:
    return load().sv_status_string(int(st)).decode()


def last_error() -> str:
    return load().sv_last_error().decode()


def _check(st: int):
    if st != SV_OK:
        raise SpecVerifyError(st, last_error())


def _ptr(t) -> Optional[int]:
    """Device pointer of a tensor (or None), with layout checks."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_contiguous():
        raise ValueError("tensors passed to libspecverify must be contiguous")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return SV_F32
    if t.dtype == torch.bfloat16:
        return SV_BF16
    raise ValueError(f"unsupported dtype {t.dtype}")


# ------------------------------------------------------------------------------------
# sv_alloc_budget
# ------------------------------------------------------------------------------------
def budget_desc(R: int, b: int, mode: str = "cost", fixed_budget: int = 0,
                ratios_pm: Sequence[int] = (250, 500, 750, 1000), cost: Sequence[int] = ()) -> BudgetDesc:
    d = BudgetDesc()
    d.num_reqs, d.block = R, b
    d.mode = SV_BUDGET_FIXED if mode == "fixed" else SV_BUDGET_COST
    d.fixed_budget = fixed_budget
    if d.mode == SV_BUDGET_COST:
        d.num_ratios = len(ratios_pm)
        for j, (r, c) in enumerate(zip(ratios_pm, cost)):
            d.ratio_permille[j] = int(r)
            d.cost[j] = int(c)
    return d


def alloc_budget(desc: BudgetDesc, conf, keep, qo_indptr, sel, scores=None, utility=None, stream=None):
    """sv_alloc_budget on torch device tensors (conf [R, b-1] fp32; outputs int32 /
    fp32 / int64-for-uint64)."""
    st = load().sv_alloc_budget(ctypes.byref(desc), _ptr(conf), _ptr(keep), _ptr(qo_indptr), _ptr(sel),
                                _ptr(scores), _ptr(utility), _stream(stream))
    _check(st)


# ------------------------------------------------------------------------------------
# sv_verify_attn
# ------------------------------------------------------------------------------------
def attn_desc(R, total_q_max, block, Hq, Hkv, d, page_size, max_pages_per_req, num_pages, max_kv_len,
              dtype: int, sm_scale: float = 0.0, kv_split: int = 0) -> AttnDesc:
    a = AttnDesc()
    (a.num_reqs, a.total_q_max, a.block, a.num_q_heads, a.num_kv_heads, a.head_dim, a.page_size,
     a.max_pages_per_req, a.num_pages, a.max_kv_len, a.dtype) = (R, total_q_max, block, Hq, Hkv, d, page_size,
                                                                 max_pages_per_req, num_pages, max_kv_len, dtype)
    a.sm_scale = sm_scale
    a.kv_split = kv_split
    return a


def attn_workspace_size(desc: AttnDesc) -> int:
    return int(load().sv_verify_attn_workspace_size(ctypes.byref(desc)))


def verify_attn(desc: AttnDesc, q, k_cache, v_cache, page_table, qo_indptr, kv_lens, out, lse=None,
                ws=None, stream=None):
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    st = load().sv_verify_attn(ctypes.byref(desc), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(page_table),
                               _ptr(qo_indptr), _ptr(kv_lens), _ptr(out), _ptr(lse), _ptr(ws), nbytes,
                               _stream(stream))
    _check(st)


def verify_attn_plan(desc: AttnDesc, qo_indptr, kv_lens, ws=None, stream=None):
    """sv_verify_attn_plan: the work plan of the bf16 path into ws."""
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    st = load().sv_verify_attn_plan(ctypes.byref(desc), _ptr(qo_indptr), _ptr(kv_lens), _ptr(ws), nbytes,
                                    _stream(stream))
    _check(st)


def verify_attn_run(desc: AttnDesc, q, k_cache, v_cache, page_table, qo_indptr, kv_lens, out, lse=None,
                    ws=None, stream=None):
    """sv_verify_attn_run: sv_verify_attn on the plan that ws holds."""
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    st = load().sv_verify_attn_run(ctypes.byref(desc), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(page_table),
                                   _ptr(qo_indptr), _ptr(kv_lens), _ptr(out), _ptr(lse), _ptr(ws), nbytes,
                                   _stream(stream))
    _check(st)


def prepare_round(bdesc: BudgetDesc, conf, keep, qo_indptr, sel, scores, utility, pdesc, block_tokens, ctx_lens,
                  tokens, positions, kv_lens, adesc=None, attn_ws=None, stream=None):
    """sv_prepare_round: budget, packing and (adesc given) the attention work plan in one launch."""
    nbytes = 0 if attn_ws is None else attn_ws.numel() * attn_ws.element_size()
    st = load().sv_prepare_round(ctypes.byref(bdesc), _ptr(conf), _ptr(keep), _ptr(qo_indptr), _ptr(sel),
                                 _ptr(scores), _ptr(utility), ctypes.byref(pdesc), _ptr(block_tokens),
                                 _ptr(ctx_lens), _ptr(tokens), _ptr(positions), _ptr(kv_lens),
                                 None if adesc is None else ctypes.byref(adesc), _ptr(attn_ws), nbytes,
                                 _stream(stream))
    _check(st)


# ------------------------------------------------------------------------------------
# sv_pack_verify / sv_append_kv
# ------------------------------------------------------------------------------------
def pack_desc(R: int, b: int, total_max: int) -> PackDesc:
    d = PackDesc()
    d.num_reqs, d.block, d.total_max = R, b, total_max
    return d


def pack_verify(desc: PackDesc, block_tokens, ctx_lens, qo_indptr, tokens, positions, kv_lens, stream=None):
    st = load().sv_pack_verify(ctypes.byref(desc), _ptr(block_tokens), _ptr(ctx_lens), _ptr(qo_indptr),
                               _ptr(tokens), _ptr(positions), _ptr(kv_lens), _stream(stream))
    _check(st)


def append_desc(R: int, total_max: int, block: int, Hkv: int, d: int, page_size: int, max_pages_per_req: int,
                num_pages: int, dtype: int) -> AppendDesc:
    a = AppendDesc()
    a.num_reqs, a.total_max, a.block, a.num_kv_heads, a.head_dim = R, total_max, block, Hkv, d
    a.page_size, a.max_pages_per_req, a.num_pages, a.dtype = page_size, max_pages_per_req, num_pages, dtype
    return a


def append_kv(desc: AppendDesc, k_new, v_new, page_table, qo_indptr, ctx_lens, k_cache, v_cache, stream=None):
    st = load().sv_append_kv(ctypes.byref(desc), _ptr(k_new), _ptr(v_new), _ptr(page_table), _ptr(qo_indptr),
                             _ptr(ctx_lens), _ptr(k_cache), _ptr(v_cache), _stream(stream))
    _check(st)


# ------------------------------------------------------------------------------------
# sv_spec_accept
# ------------------------------------------------------------------------------------
def accept_desc(R: int, b: int, V: int, kind: int, dtype: int, temperature: float = 1.0) -> AcceptDesc:
    a = AcceptDesc()
    a.num_reqs, a.block, a.vocab, a.kind, a.dtype = R, b, V, kind, dtype
    a.temperature = temperature
    return a


def accept_workspace_size(desc: AcceptDesc) -> int:
    return int(load().sv_spec_accept_workspace_size(ctypes.byref(desc)))


def spec_accept(desc: AcceptDesc, target, draft, draft_tokens, qo_indptr, u_accept, u_sample, accept_len,
                out_tokens, flags=None, ws=None, stream=None):
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    st = load().sv_spec_accept(ctypes.byref(desc), _ptr(target), _ptr(draft), _ptr(draft_tokens),
                               _ptr(qo_indptr), _ptr(u_accept), _ptr(u_sample), _ptr(accept_len),
                               _ptr(out_tokens), _ptr(flags), _ptr(ws), nbytes, _stream(stream))
    _check(st)


def spec_accept_noalloc(desc: AcceptDesc, target, draft, draft_tokens, qo_indptr, u_accept, u_sample, accept_len,
                        out_tokens, flags=None, stream=None):
    """sv_spec_accept_noalloc: the library's fixed device scratch replaces the workspace."""
    st = load().sv_spec_accept_noalloc(ctypes.byref(desc), _ptr(target), _ptr(draft), _ptr(draft_tokens),
                                       _ptr(qo_indptr), _ptr(u_accept), _ptr(u_sample), _ptr(accept_len),
                                       _ptr(out_tokens), _ptr(flags), _stream(stream))
    _check(st)


def spec_accept_debug(desc: AcceptDesc, target, draft, draft_tokens, qo_indptr, u_accept, u_sample, accept_len,
                      out_tokens, flags, dbg_pq, dbg_row, ws=None, stream=None):
    """sv_spec_accept_debug: sv_spec_accept plus the fp32 values its decisions were taken on."""
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    st = load().sv_spec_accept_debug(ctypes.byref(desc), _ptr(target), _ptr(draft), _ptr(draft_tokens),
                                     _ptr(qo_indptr), _ptr(u_accept), _ptr(u_sample), _ptr(accept_len),
                                     _ptr(out_tokens), _ptr(flags), _ptr(dbg_pq), _ptr(dbg_row), _ptr(ws), nbytes,
                                     _stream(stream))
    _check(st)


# ------------------------------------------------------------------------------------
# sv_spec_accept_stats, sv_draft_stats
# ------------------------------------------------------------------------------------
def spec_accept_stats(desc: AcceptDesc, target, draft, draft_stats, draft_tokens, qo_indptr, u_accept, u_sample,
                      accept_len, out_tokens, flags=None, ws=None, stream=None):
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    st = load().sv_spec_accept_stats(ctypes.byref(desc), _ptr(target), _ptr(draft), _ptr(draft_stats),
                                     _ptr(draft_tokens), _ptr(qo_indptr), _ptr(u_accept), _ptr(u_sample),
                                     _ptr(accept_len), _ptr(out_tokens), _ptr(flags), _ptr(ws), nbytes,
                                     _stream(stream))
    _check(st)


def draft_stats_desc(R: int, drafts: int, V: int, dtype: int, temperature: float = 1.0) -> DraftStatsDesc:
    d = DraftStatsDesc()
    d.num_reqs, d.drafts, d.vocab, d.dtype, d.temperature = R, drafts, V, dtype, temperature
    return d


def draft_stats_workspace_size(desc: DraftStatsDesc) -> int:
    return int(load().sv_draft_stats_workspace_size(ctypes.byref(desc)))


def draft_stats(desc: DraftStatsDesc, draft_logits, stats, conf=None, ws=None, stream=None):
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    st = load().sv_draft_stats(ctypes.byref(desc), _ptr(draft_logits), _ptr(stats), _ptr(conf), _ptr(ws), nbytes,
                               _stream(stream))
    _check(st)
