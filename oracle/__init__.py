"""CPU oracle for the draft-verify round: test infrastructure only.

Plain C (oracle.c), loaded with ctypes and driven with numpy arrays. Only the
test-suite, the smoke check and the CPU-baseline leg of the benchmark use it; the
GPU library never loads or calls it and shares no code with it.

Every function follows one passage of the paper (AngelSpec):
  budget()       -- D-cut, Sec. 4.2: eqs. dcut-score, dcut-budget,
                    dcut-batch-utility, dcut-select and the packing paragraph.
  accept()       -- rejection-sampling verification (Sec. 1; overlap identity
                    eq. mtp-acceptance-tv), with the extra token drawn from the
                    residual max(p-q, 0) or, when every draft survives, from p.
  attention()    -- verify attention of every kept position (Sec. 4.1-4.2),
                    written out as the dense masked softmax definition in fp64.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# SV_ORACLE_LIB names another build of oracle.c (the sanitizer test loads an
# AddressSanitizer/UndefinedBehaviorSanitizer build through it)
_LIB_PATH = os.environ.get("SV_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i32 = ctypes.c_int
    lib.oracle_prefix_scores.argtypes = [i32, i32, P, P]
    lib.oracle_prefix_scores.restype = None
    lib.oracle_budget.argtypes = [i32, i32, i32, i32, i32, P, P, P, P, P, P, P, P]
    lib.oracle_budget.restype = i32
    lib.oracle_accept.argtypes = [i32, i32, i32, i32, i32, ctypes.c_float, P, P, P, P, P, P,
                                  P, P, P, P, P, P]
    lib.oracle_accept.restype = i32
    lib.oracle_accept_greedy.argtypes = [i32, i32, i32, i32, P, P, P, P, P, P]
    lib.oracle_accept_greedy.restype = i32
    lib.oracle_attn.argtypes = [i32, i32, i32, i32, i32, i32, i32, i32, P, P, P, P, P, P,
                                ctypes.c_double, i32, P, P, P, P]
    lib.oracle_attn.restype = i32
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = i32
    lib.oracle_set_num_threads.argtypes = [i32]
    lib.oracle_set_num_threads.restype = i32
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> int:
    """Threads of the oracle's parallel loops from now on; returns the new setting."""
    return int(_load().oracle_set_num_threads(int(n)))


def prefix_scores(conf: np.ndarray) -> np.ndarray:
    """eq. dcut-score: [R, b-1] confidences -> [R, b] fp32 prefix products."""
    conf = _c(conf, np.float32)
    R, D = conf.shape
    out = np.empty((R, D + 1), np.float32)
    _load().oracle_prefix_scores(R, D + 1, _ptr(conf), _ptr(out))
    return out


def budget(conf, mode="cost", fixed_budget=0, ratios_pm=(250, 500, 750, 1000), cost=None):
    """D-cut budget (Sec. 4.2). conf [R, b-1] fp32.

    mode "fixed": keep the top `fixed_budget` positions; mode "cost": pick
    rho* = argmax U/C over `ratios_pm` (permille) with `cost` = C(R, rho_j).
    Returns dict(keep [R], qo_indptr [R+1], K, rho_index, scores [R,b], utility).
    """
    conf = _c(conf, np.float32)
    R, D = conf.shape
    b = D + 1
    m = 0 if mode == "fixed" else 1
    nr = len(ratios_pm)
    rp = _c(list(ratios_pm) + [0] * (8 - nr), np.int32)
    cst = _c(list(cost if cost is not None else [1] * nr) + [0] * (8 - nr), np.uint32)
    keep = np.empty(R, np.int32)
    qo = np.empty(R + 1, np.int32)
    sel = np.empty(2, np.int32)
    scores = np.empty((R, b), np.float32)
    util = np.zeros(max(nr, 1), np.uint64)
    rc = _load().oracle_budget(R, b, m, int(fixed_budget), nr, _ptr(rp), _ptr(cst), _ptr(conf),
                               _ptr(keep), _ptr(qo), _ptr(sel), _ptr(scores), _ptr(util))
    if rc != 0:
        raise ValueError("oracle_budget: invalid arguments")
    return dict(keep=keep, qo_indptr=qo, K=int(sel[0]), rho_index=int(sel[1]), scores=scores,
                utility=util if m == 1 else util[:1])


def accept(target, draft, draft_tokens, qo_indptr, u_accept, u_sample, kind="probs",
           dtype="f32", temperature=1.0, diagnostics=False):
    """Speculative acceptance for R requests (see oracle.c for the exact steps).

    target [K, V] packed rows (fp32, or uint16 bf16 bits when dtype="bf16");
    draft [R, b-1, V]; draft_tokens [R, b-1] int32; qo_indptr [R+1];
    u_accept [R, b-1] fp32; u_sample [R] fp32.
    Returns dict(accept_len [R], out_tokens [R, b], flags [R]) and, with
    diagnostics, p_at/q_at [R, b-1] and cdf [R, 4] = (thr, cum before token, token weight, Z).
    """
    dt = 0 if dtype == "f32" else 1
    knd = 1 if kind == "probs" else 0
    edt = np.float32 if dt == 0 else np.uint16
    target = _c(target, edt)
    if temperature == 0:
        return accept_greedy(target, np.asarray(draft).shape, draft_tokens, qo_indptr, dtype)
    draft = _c(draft, edt)
    R, D, V = draft.shape
    b = D + 1
    dtok = _c(draft_tokens, np.int32).reshape(R, D)
    qo = _c(qo_indptr, np.int32)
    ua = _c(u_accept, np.float32).reshape(R, D)
    us = _c(u_sample, np.float32).reshape(R)
    acc = np.empty(R, np.int32)
    out = np.empty((R, b), np.int32)
    flags = np.empty(R, np.int32)
    dp = np.zeros((R, D), np.float64) if diagnostics else None
    dq = np.zeros((R, D), np.float64) if diagnostics else None
    dc = np.zeros((R, 4), np.float64) if diagnostics else None
    rc = _load().oracle_accept(R, b, V, knd, dt, float(temperature), _ptr(target), _ptr(draft),
                               _ptr(dtok), _ptr(qo), _ptr(ua), _ptr(us), _ptr(acc), _ptr(out),
                               _ptr(flags), _ptr(dp), _ptr(dq), _ptr(dc))
    if rc != 0:
        raise ValueError("oracle_accept: invalid arguments")
    res = dict(accept_len=acc, out_tokens=out, flags=flags)
    if diagnostics:
        res.update(p_at=dp, q_at=dq, cdf=dc)
    return res


def accept_greedy(target, draft_shape, draft_tokens, qo_indptr, dtype="f32"):
    """Greedy verification (temperature 0, see oracle.c): argmax of each target row,
    lowest index on ties, NaN skipped. draft_shape = (R, b-1, V) (draft rows are not
    read). Returns dict(accept_len, out_tokens, flags)."""
    dt = 0 if dtype == "f32" else 1
    edt = np.float32 if dt == 0 else np.uint16
    target = _c(target, edt)
    R, D, V = draft_shape
    b = D + 1
    dtok = _c(draft_tokens, np.int32).reshape(R, D)
    qo = _c(qo_indptr, np.int32)
    acc = np.empty(R, np.int32)
    out = np.empty((R, b), np.int32)
    flags = np.empty(R, np.int32)
    rc = _load().oracle_accept_greedy(R, b, V, dt, _ptr(target), _ptr(dtok), _ptr(qo), _ptr(acc), _ptr(out),
                                      _ptr(flags))
    if rc != 0:
        raise ValueError("oracle_accept_greedy: invalid arguments")
    return dict(accept_len=acc, out_tokens=out, flags=flags)


def attention(q, k_cache, v_cache, page_table, qo_indptr, kv_lens, scale=None, dtype="f32",
              units=None):
    """Dense verify attention in fp64.

    q [K, Hq, d]; k_cache/v_cache [num_pages, Hkv, P, d]; page_table [R, maxp];
    qo_indptr [R+1]; kv_lens [R] (= committed context + k_i). dtype "bf16" means
    the arrays hold uint16 bf16 bits. units: None for every (row, head), else a
    pair of int arrays (rows, heads). Returns (out [n, d] fp64, lse [n] fp64).
    """
    dt = 0 if dtype == "f32" else 1
    edt = np.float32 if dt == 0 else np.uint16
    q = _c(q, edt)
    kc = _c(k_cache, edt)
    vc = _c(v_cache, edt)
    K, Hq, d = q.shape
    num_pages, Hkv, P, d2 = kc.shape
    assert d2 == d and vc.shape == kc.shape
    pt = _c(page_table, np.int32)
    R, maxp = pt.shape
    qo = _c(qo_indptr, np.int32)
    kl = _c(kv_lens, np.int32)
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    if units is None:
        n = K * Hq
        rows = heads = None
        nsel = -1
    else:
        rows = _c(units[0], np.int32)
        heads = _c(units[1], np.int32)
        n = nsel = len(rows)
    out = np.empty((n, d), np.float64)
    lse = np.empty(n, np.float64)
    rc = _load().oracle_attn(R, Hq, Hkv, d, P, maxp, num_pages, dt, _ptr(q), _ptr(kc), _ptr(vc),
                             _ptr(pt), _ptr(qo), _ptr(kl), float(scale), nsel, _ptr(rows),
                             _ptr(heads), _ptr(out), _ptr(lse))
    if rc != 0:
        raise ValueError("oracle_attn: invalid arguments")
    return out, lse


# ------------------------------------------------------------------------------------
# packing of the verify batch and the cache append (Sec. 4.2, "Packing and correctness")
# ------------------------------------------------------------------------------------
def pack_verify(block_tokens, ctx_lens, qo_indptr, total_max):
    """Dense verify batch: row qo[i] + j (j < k_i) holds block_tokens[i][j] at absolute
    position ctx_lens[i] + j; kv_lens[i] = ctx_lens[i] + k_i. A request with k_i outside
    [1, b] or rows outside [0, total_max) gets no rows and kv_lens[i] = ctx_lens[i].
    Returns (tokens, positions, kv_lens); unwritten rows hold -1."""
    bt = np.asarray(block_tokens, np.int32)
    R, b = bt.shape
    L = np.asarray(ctx_lens, np.int64)
    qo = np.asarray(qo_indptr, np.int64)
    tokens = np.full(total_max, -1, np.int32)
    positions = np.full(total_max, -1, np.int32)
    kv_lens = np.zeros(R, np.int32)
    for i in range(R):
        k = int(qo[i + 1] - qo[i])
        ok = 1 <= k <= b and qo[i] >= 0 and qo[i] + k <= total_max
        kv_lens[i] = L[i] + k if ok else L[i]
        if not ok:
            continue
        for j in range(k):
            tokens[qo[i] + j] = bt[i, j]
            positions[qo[i] + j] = L[i] + j
    return tokens, positions, kv_lens


def append_kv(k_new, v_new, page_table, qo_indptr, ctx_lens, k_cache, v_cache, block):
    """Copies of the caches with row qo[i] + j of k_new / v_new (every kv-head) written at
    position s = ctx_lens[i] + j: page page_table[i][s // P], slot s % P. Rows of a request
    with k_i outside [1, block], or whose page column or page id is out of range, are
    skipped."""
    kc = np.array(k_cache, copy=True)
    vc = np.array(v_cache, copy=True)
    num_pages, Hkv, P, d = kc.shape
    pt = np.asarray(page_table)
    R, maxp = pt.shape
    qo = np.asarray(qo_indptr, np.int64)
    total = np.asarray(k_new).shape[0]
    for i in range(R):
        k = int(qo[i + 1] - qo[i])
        if not (1 <= k <= block and qo[i] >= 0 and qo[i] + k <= total) or ctx_lens[i] < 0:
            continue
        for j in range(k):
            s = int(ctx_lens[i]) + j
            col = s // P
            if col >= maxp:
                continue
            pg = int(pt[i, col])
            if pg < 0 or pg >= num_pages:
                continue
            kc[pg, :, s % P, :] = k_new[qo[i] + j]
            vc[pg, :, s % P, :] = v_new[qo[i] + j]
    return kc, vc


# ------------------------------------------------------------------------------------
# draft-row statistics (the confidence c_t of Sec. 4.2 and the draft softmax normaliser)
# ------------------------------------------------------------------------------------
def draft_stats(draft_logits, temperature=1.0, dtype="f32"):
    """For every draft row (last axis = vocabulary) of the stored logits l (fp32, or
    uint16 bf16 bits when dtype="bf16"), in fp64: m = max_v l(v)/T,
    S = sum_v exp(l(v)/T - m), conf = max_v softmax(l/T)(v) = 1/S.
    Returns dict(m, S, conf) shaped like the rows."""
    x = np.asarray(draft_logits)
    if dtype == "bf16":
        x = (x.astype(np.uint32) << 16).view(np.float32)
    z = x.astype(np.float64) / float(np.float32(temperature))
    m = z.max(axis=-1)
    S = np.exp(z - m[..., None]).sum(axis=-1)
    return dict(m=m, S=S, conf=1.0 / S)
