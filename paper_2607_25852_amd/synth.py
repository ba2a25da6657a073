"""Seeded synthetic inputs for one draft-verify round.

This module plays the parts of the system that sit *outside* the verify path:
the drafter (draft logits, its sampled tokens and per-position confidences), the
target model (target logits / probabilities, queries, paged KV cache), the
serving scheduler (committed context lengths, page allocation) and the
start-up profiler (a cost table). It holds none of the verify path's
arithmetic; both the GPU library's tests and the CPU oracle consume what it
makes.

Shapes follow the serving workloads of the paper's deployment experiments
(concurrency 4-64, draft blocks of 8 or 16 positions, MTP depth 4, vocabularies
up to 131072); the public benchmarks themselves are not reproduced, random
draws of matching shape stand in for them.

Every draw uses its own counter-addressed numpy stream
``default_rng([seed, stream, index])`` so a single request's rows can be made
again on their own, e.g. to check a sampled output of a full-size run.
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional

import numpy as np

# stream ids of the counter-addressed generators
_S_TARGET, _S_DRAFT, _S_CLASS, _S_TOK, _S_UACC, _S_USMP, _S_KVLEN, _S_PAGES, _S_K, _S_V, _S_Q, \
    _S_KSEL, _S_PEAK = range(13)

# per-request difficulty classes: (draft noise sigma, range of the target's peak mass)
CLASSES = ((0.3, 0.85, 0.999), (1.0, 0.40, 0.95), (2.0, 0.02, 0.50))
PAPER_RATIOS_PM = (250, 500, 750, 1000)  # {0.25, 0.5, 0.75, 1.0}, Sec. 4.2
COST_A_US, COST_B_US, COST_C_US = 20000, 15, 2000  # synthetic profile: a + b*tok + c*ceil(tok/256)


def _rng(seed: int, stream: int, index: int = 0) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(stream), int(index)])


# ---------------------------------------------------------------------------
# encodings
# ---------------------------------------------------------------------------
def bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even; NaN stays NaN."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    t = (u >> 16) & 1
    t += u
    t += 0x7FFF  # wraps only for NaN bit patterns, which are replaced below
    t >>= 16
    rounded = t.astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        rounded[nan] = 0x7FC0
    return rounded


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def uniforms_24(rng: np.random.Generator, shape) -> np.ndarray:
    """Uniforms in [0, 1) on the 2^-24 grid, as fp32 (exact)."""
    return (rng.integers(0, 1 << 24, size=shape, dtype=np.int64).astype(np.float64)
            * 2.0 ** -24).astype(np.float32)


# ---------------------------------------------------------------------------
# workload descriptions
# ---------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class RoundConfig:
    name: str
    R: int                 # concurrent requests
    b: int                 # block positions per request (certain token + D drafts)
    V: int                 # vocabulary
    dtype: str             # "f32" | "bf16" for logits, q and KV
    Hq: int
    Hkv: int
    d: int
    page: int
    kv: tuple              # ("list", L...) | ("uniform", lo, hi) | ("lognormal", median, sigma, lo, hi)
    logits: tuple          # ("plain", target_sigma, draft_sigma) | ("classes",) | ("class", k)
    budget: tuple          # ("fixed", K) | ("cost",) | ("given",)  (k_i ~ U{1..b}, no budget step)
    seed: int

    @property
    def D(self) -> int:
        return self.b - 1


def _cfgs():
    c = {}
    c["tiny"] = RoundConfig("tiny", 4, 8, 1024, "f32", 8, 2, 64, 16, ("list", 37, 128, 255, 512),
                            ("plain", 2.0, 0.5), ("fixed", 32), 1234)
    c["c16_b16"] = RoundConfig("c16_b16", 16, 16, 32768, "bf16", 32, 8, 128, 64,
                               ("uniform", 1024, 8192), ("plain", 3.0, 1.0), ("fixed", 256), 1235)
    c["c64_b16"] = RoundConfig("c64_b16", 64, 16, 131072, "bf16", 64, 8, 128, 64,
                               ("lognormal", 4096, 1.0, 512, 32768), ("classes",), ("cost",), 1236)
    c["long_c32"] = RoundConfig("long_c32", 32, 16, 131072, "bf16", 64, 4, 128, 64,
                                ("uniform", 65536, 131072), ("class", 1), ("given",), 1237)
    for R in (4, 8, 16, 32, 64):
        for b, mode in ((5, "mtp"), (16, "blk")):
            c[f"sweep_{mode}_c{R}"] = RoundConfig(
                f"sweep_{mode}_c{R}", R, b, 131072, "bf16", 64, 8, 128, 64,
                ("lognormal", 8192, 1.0, 512, 65536), ("classes",), ("cost",), 1238)
    return c


CONFIGS = _cfgs()


# ---------------------------------------------------------------------------
# committed context and verify depth
# ---------------------------------------------------------------------------
def kv_context_lengths(cfg: RoundConfig) -> np.ndarray:
    """Committed context length L_i per request (tokens before the verify block)."""
    kind = cfg.kv[0]
    g = _rng(cfg.seed, _S_KVLEN)
    if kind == "list":
        L = np.array(cfg.kv[1:], dtype=np.int64)
        assert len(L) == cfg.R
    elif kind == "uniform":
        L = g.integers(cfg.kv[1], cfg.kv[2] + 1, size=cfg.R)
    elif kind == "lognormal":
        med, sig, lo, hi = cfg.kv[1:]
        L = np.clip(np.round(np.exp(g.normal(math.log(med), sig, size=cfg.R))), lo, hi)
    else:
        raise ValueError(kind)
    return L.astype(np.int32)


def given_depths(cfg: RoundConfig) -> np.ndarray:
    """Verify depths k_i ~ U{1..b} for workloads that skip the budget step."""
    return _rng(cfg.seed, _S_KSEL).integers(1, cfg.b + 1, size=cfg.R).astype(np.int32)


def indptr_from_depths(k: np.ndarray) -> np.ndarray:
    qo = np.zeros(len(k) + 1, np.int32)
    qo[1:] = np.cumsum(k)
    return qo


# ---------------------------------------------------------------------------
# logits, probabilities, draft tokens, confidences
# ---------------------------------------------------------------------------
def request_class(cfg: RoundConfig, i: int) -> Optional[int]:
    """Difficulty class of request i: a seeded shuffle of a balanced round-robin
    over the three classes (so every batch mixes them in equal shares)."""
    if cfg.logits[0] == "classes":
        return int(_rng(cfg.seed, _S_CLASS).permutation(np.arange(cfg.R) % 3)[i])
    if cfg.logits[0] == "class":
        return int(cfg.logits[1])
    return None


def _softmax64(x: np.ndarray) -> np.ndarray:
    """fp64 softmax used only to *produce* inputs (the model side)."""
    z = x.astype(np.float64)
    z = z - z.max(axis=-1, keepdims=True)
    e = np.exp(z)
    return e / e.sum(axis=-1, keepdims=True)


def request_logits(cfg: RoundConfig, i: int):
    """fp32 logits of request i: target [b, V] (row r = position r+1) and draft [D, V]
    (row t-1 = draft t), before any bf16 encoding."""
    V, b, D = cfg.V, cfg.b, cfg.D
    kind = cfg.logits[0]
    gt = _rng(cfg.seed, _S_TARGET, i)
    gd = _rng(cfg.seed, _S_DRAFT, i)
    if kind == "plain":
        ts, ds = cfg.logits[1], cfg.logits[2]
        tgt = gt.standard_normal((b, V), dtype=np.float32) * np.float32(ts)
        noise = gd.standard_normal((D, V), dtype=np.float32) * np.float32(ds)
        dft = tgt[:D] + noise
        return tgt, dft
    k = request_class(cfg, i)
    sigma, lo, hi = CLASSES[k]
    tgt = gt.standard_normal((b, V), dtype=np.float32) * np.float32(3.0)
    gp = _rng(cfg.seed, _S_PEAK, i)
    peak_tok = gp.integers(0, V, size=b)
    peak_mass = gp.uniform(lo, hi, size=b)
    for r in range(b):
        rest = np.delete(tgt[r].astype(np.float64), peak_tok[r])
        m = rest.max()
        lse_rest = m + math.log(np.exp(rest - m).sum())
        tgt[r, peak_tok[r]] = np.float32(math.log(peak_mass[r] / (1.0 - peak_mass[r])) + lse_rest)
    noise = gd.standard_normal((D, V), dtype=np.float32) * np.float32(sigma)
    dft = tgt[:D] + noise
    return tgt, dft


def encode(cfg: RoundConfig, x: np.ndarray) -> np.ndarray:
    """Storage form of a float array for this workload: fp32, or bf16 bits."""
    return np.ascontiguousarray(x, np.float32) if cfg.dtype == "f32" else bf16_bits(x)


def stored_as_f32(cfg: RoundConfig, x: np.ndarray) -> np.ndarray:
    """The fp32 value of what is stored (bf16 rounding applied when the workload is bf16)."""
    return np.ascontiguousarray(x, np.float32) if cfg.dtype == "f32" else bf16_to_f32(bf16_bits(x))


def draft_side(cfg: RoundConfig, i: int, dft_stored_f32: np.ndarray):
    """The drafter's own outputs for request i: tokens d_t sampled from its
    distribution q_t = softmax(draft logits) and the confidence c_t = max_v q_t(v)
    (the confidence definition of the block-diffusion sweep workloads)."""
    q = _softmax64(dft_stored_f32)
    u = _rng(cfg.seed, _S_TOK, i).random(cfg.D)
    cdf = np.cumsum(q, axis=-1)
    tok = np.array([min(int(np.searchsorted(cdf[t], u[t] * cdf[t, -1], side="right")), cfg.V - 1)
                    for t in range(cfg.D)], dtype=np.int32)
    conf = q.max(axis=-1).astype(np.float32)
    return tok, conf


def make_logits_round(cfg: RoundConfig, want_probs: bool = False, requests=None):
    """Target rows for every block position, draft rows, draft tokens, confidences.

    Returns a dict with
      target_full [R, b, V]  (storage dtype: fp32 or uint16 bf16 bits)
      draft       [R, D, V]  (storage dtype)
      draft_tokens [R, D] int32, conf [R, D] fp32,
      and, with want_probs, target_probs_full [R, b, V] / draft_probs [R, D, V] fp32
      (the probability rows a sampler would hand over: fp64 softmax of the
      stored logits, rounded to fp32).
    """
    reqs = range(cfg.R) if requests is None else requests
    n = len(reqs)
    st = np.float32 if cfg.dtype == "f32" else np.uint16
    tfull = np.empty((n, cfg.b, cfg.V), st)
    dft = np.empty((n, cfg.D, cfg.V), st)
    toks = np.empty((n, cfg.D), np.int32)
    conf = np.empty((n, cfg.D), np.float32)
    tp = np.empty((n, cfg.b, cfg.V), np.float32) if want_probs else None
    dp = np.empty((n, cfg.D, cfg.V), np.float32) if want_probs else None
    def one(k_i):
        k, i = k_i
        t32, d32 = request_logits(cfg, i)
        tfull[k] = encode(cfg, t32)
        dft[k] = encode(cfg, d32)
        d_stored = stored_as_f32(cfg, d32)
        toks[k], conf[k] = draft_side(cfg, i, d_stored)
        if want_probs:
            tp[k] = _softmax64(stored_as_f32(cfg, t32)).astype(np.float32)
            dp[k] = _softmax64(d_stored).astype(np.float32)

    # every request has its own generators: parallel filling equals sequential filling
    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        list(ex.map(one, enumerate(reqs)))
    out = dict(target_full=tfull, draft=dft, draft_tokens=toks, conf=conf)
    if want_probs:
        out.update(target_probs_full=tp, draft_probs=dp)
    return out


def acceptance_uniforms(cfg: RoundConfig):
    """u_accept [R, D] and u_sample [R], on the 2^-24 grid."""
    ua = np.stack([uniforms_24(_rng(cfg.seed, _S_UACC, i), cfg.D) for i in range(cfg.R)])
    us = np.array([uniforms_24(_rng(cfg.seed, _S_USMP, i), 1)[0] for i in range(cfg.R)],
                  dtype=np.float32)
    return ua.astype(np.float32).reshape(cfg.R, cfg.D), us


def pack_rows(full: np.ndarray, qo_indptr: np.ndarray) -> np.ndarray:
    """Rows 0..k_i-1 of every request, packed densely in request order (the rows
    the target model would have produced for the kept positions)."""
    k = np.diff(qo_indptr)
    parts = [full[i, :k[i]] for i in range(full.shape[0])]
    return np.ascontiguousarray(np.concatenate(parts, axis=0))


# ---------------------------------------------------------------------------
# start-up cost profile (a stand-in for profiling C(B, rho) on a real server)
# ---------------------------------------------------------------------------
def profiled_cost(R: int, b: int, ratios_pm=PAPER_RATIOS_PM, a=COST_A_US, per_tok=COST_B_US,
                  step=COST_C_US) -> np.ndarray:
    """Synthetic step latency in microseconds for each ratio at batch R: a server whose
    step time is a + per_tok*tok + step*ceil(tok/256) when it verifies tok positions
    (tok = the budget that ratio allows: at least one position per request)."""
    out = []
    for pm in ratios_pm:
        tok = max(R, -(-pm * R * b // 1000))
        out.append(a + per_tok * tok + step * (-(-tok // 256)))
    return np.array(out, dtype=np.uint32)


# ---------------------------------------------------------------------------
# queries and paged KV cache
# ---------------------------------------------------------------------------
def make_kv(cfg: RoundConfig, L: np.ndarray, fill_unused=0.0, pool_slack=1.25, q_scale=1.0,
            zero_k=False, want_cache=True):
    """Queries for every block position and a paged cache holding L_i + b tokens
    per request (the block's own K/V already written after the context).

    Pages of request i are drawn without replacement from a pool `pool_slack`
    times larger than needed (a shuffled page table); pool pages nobody owns and
    slots past a request's last token hold `fill_unused` (NaN in poison tests).
    Returns dict(q_full [R, b, Hq, d], k_cache, v_cache [num_pages, Hkv, P, d],
    page_table [R, maxp] int32) in storage dtype.
    """
    R, b, P, Hkv, Hq, d = cfg.R, cfg.b, cfg.page, cfg.Hkv, cfg.Hq, cfg.d
    need = [(-(-(int(L[i]) + b) // P)) for i in range(R)]
    maxp = max(need)
    pool = int(math.ceil(sum(need) * pool_slack))
    perm = _rng(cfg.seed, _S_PAGES).permutation(pool).astype(np.int32)
    pt = np.full((R, maxp), -1, np.int32)
    cur = 0
    for i in range(R):
        pt[i, :need[i]] = perm[cur:cur + need[i]]
        cur += need[i]
    st = np.float32 if cfg.dtype == "f32" else np.uint16
    gq = _rng(cfg.seed, _S_Q)
    q32 = gq.standard_normal((R, b, Hq, d), dtype=np.float32) * np.float32(q_scale)
    out = dict(q_full=encode(cfg, q32), page_table=pt, num_pages=pool)
    if not want_cache:
        return out
    fill = encode(cfg, np.array([fill_unused], np.float32))[0]
    kc = np.full((pool, Hkv, P, d), fill, st)
    vc = np.full((pool, Hkv, P, d), fill, st)

    def fill(i):
        ntok = int(L[i]) + b
        kk = _rng(cfg.seed, _S_K, i).standard_normal((Hkv, ntok, d), dtype=np.float32)
        vv = _rng(cfg.seed, _S_V, i).standard_normal((Hkv, ntok, d), dtype=np.float32)
        if zero_k:
            kk[:] = 0.0
        kk = encode(cfg, kk)
        vv = encode(cfg, vv)
        for p in range(need[i]):
            lo = p * P
            cnt = min(P, ntok - lo)
            kc[pt[i, p], :, :cnt] = kk[:, lo:lo + cnt]
            vc[pt[i, p], :, :cnt] = vv[:, lo:lo + cnt]

    # requests own disjoint pages and their own generators: filling them in parallel
    # gives the same cache as filling them in order
    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        list(ex.map(fill, range(R)))
    out.update(k_cache=kc, v_cache=vc)
    return out
