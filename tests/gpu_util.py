"""Helpers shared by the GPU parity tests (marshalling, cached inputs and comparison only)."""
import functools
import sys

import numpy as np

SWEEP = [f"sweep_{m}_c{r}" for m in ("mtp", "blk") for r in (4, 8, 16, 32, 64)]
_CONF = {}


@functools.lru_cache(maxsize=2)
def logits_round(name, want_probs=False):
    """The generator's logits round of a named workload (the last two are kept: tests of
    one workload in different modes reuse them)."""
    from paper_2607_25852_amd import synth
    lr = synth.make_logits_round(synth.CONFIGS[name], want_probs=want_probs)
    _CONF[name] = lr["conf"]
    return lr


def conf_of(name):
    """The drafter's confidences of a named workload (kept for the whole session)."""
    if name not in _CONF:
        logits_round(name, False)
    return _CONF[name]


def budget_packing(name):
    """qo_indptr of a named workload as its round packs it: the budget's own choice
    (fixed or cost table, computed by the oracle) or the given depths."""
    from paper_2607_25852_amd import synth
    import oracle
    cfg = synth.CONFIGS[name]
    if cfg.budget[0] == "given":
        return synth.indptr_from_depths(synth.given_depths(cfg))
    if cfg.budget[0] == "fixed":
        return oracle.budget(conf_of(name), "fixed", fixed_budget=cfg.budget[1])["qo_indptr"]
    return oracle.budget(conf_of(name), "cost", cost=synth.profiled_cost(cfg.R, cfg.b))["qo_indptr"]


def say(*a):
    """Progress line naming the case, flushed before the GPU step it precedes."""
    print("[gpu]", *a, file=sys.stderr, flush=True)


def bf16_bits_of(t):
    """torch bf16 device tensor -> numpy uint16 bit patterns."""
    import torch
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)


def f32_of_bits(bits):
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32)


def compare_attention(out_gpu, lse_gpu, out_ref, lse_ref, dtype):
    """Tolerance gate of verify attention: max-abs 2e-2 (bf16) / 1e-5 (fp32), plus a
    relative RMS and an lse check that a near-zero output could not pass by accident."""
    out_gpu = np.asarray(out_gpu, np.float64)
    err = np.abs(out_gpu - out_ref)
    max_abs = float(err.max()) if err.size else 0.0
    rms_ref = float(np.sqrt(np.mean(out_ref ** 2))) if err.size else 1.0
    rel_rms = float(np.sqrt(np.mean(err ** 2))) / max(rms_ref, 1e-30) if err.size else 0.0
    dlse = float(np.abs(np.asarray(lse_gpu, np.float64) - lse_ref).max()) if err.size else 0.0
    if dtype == "bf16":
        ok = max_abs <= 2e-2 and rel_rms <= 1e-2 and dlse <= 1e-3
    else:
        ok = max_abs <= 1e-5 and rel_rms <= 1e-5 and dlse <= 1e-5
    return ok, dict(max_abs=max_abs, rel_rms=rel_rms, max_dlse=dlse, n=int(out_ref.shape[0]))


def classify_accept(gpu, ref, ua, rel_tol=1e-5, cdf_tol=2.0 ** -20):
    """Logits-mode comparison (the parity contract: decisions agree wherever the oracle's
    margin |u*q - p| exceeds 1e-5*p and the threshold lies more than 2^-20*Z from a CDF
    step). Returns (n_exact, n_marginal, failures): a request whose outputs differ is
    'marginal' only when the oracle's own decision sat within rel_tol of its boundary
    (acceptance) or the draw within cdf_tol*Z of a CDF step; anything else is a failure."""
    R = len(ref["accept_len"])
    exact = marginal = 0
    failures = []
    for i in range(R):
        ag, ao = int(gpu["accept_len"][i]), int(ref["accept_len"][i])
        if ag == ao and np.array_equal(gpu["out_tokens"][i], ref["out_tokens"][i]):
            exact += 1
            continue
        if ag != ao:
            t = min(ag, ao)  # 0-based index of the first draft decided differently
            p, q, u = ref["p_at"][i, t], ref["q_at"][i, t], float(ua[i, t])
            if abs(u * q - p) <= rel_tol * p:
                marginal += 1
            else:
                failures.append((i, "accept", ag, ao, p, q, u))
            continue
        thr, cb, wt, Z = ref["cdf"][i]
        if min(thr - cb, cb + wt - 1 - thr) <= cdf_tol * Z:
            marginal += 1
        else:
            failures.append((i, "token", gpu["out_tokens"][i].tolist(), ref["out_tokens"][i].tolist()))
    return exact, marginal, failures
