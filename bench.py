"""Benchmark of one draft-verify round on one MI355X.

A step is the whole round on resident inputs, on one stream, with no host round trip:
  sv_alloc_budget (D-cut: prefix scores, global top-K, cost-table ratio, packing)
  sv_pack_verify  (the verify batch's tokens and positions, and the key counts L_i + k_i)
  sv_verify_attn  (one layer of verify attention over the paged KV cache)
  sv_spec_accept  (softmax of bf16 logits, accept test, first-reject cut, residual/bonus draw)
Workload (default): concurrency 64, block 16 (15 drafts + the certain token), bf16,
64 query / 8 KV heads of dim 128, committed context lognormal (median 4096, clipped
to [512, 32768]) in 64-token pages, vocabulary 131072, per-request draft noise drawn
from {0.3, 1.0, 2.0}, budget ratio chosen by a linear-plus-step cost table.

Metric: verified draft tokens per second (sum of kept drafts n_i per step / step time).
After the main workload every other named workload is timed the same way ("workloads"),
and the CPU oracle is timed per part at one thread and at all threads on a bounded sample
of each ("cpu_baseline"). Warm-up before every timed loop: the asked-for number of steps
and at least 0.2 s of them, since the GPU's clocks settle only after about 20 ms of
sustained work. One JSON line on stdout; progress on stderr.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
ATTN_SRC = os.path.join(ROOT, "paper_2607_25852_amd", "csrc", "attn.hip")
# HBM traffic of one sv_verify_attn call, from rocprofv3 FETCH_SIZE / WRITE_SIZE runs
# scaled by a copy kernel of known size; valid only while the attention source is the
# one that was measured (its digest is recorded beside the figure)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "sv_verify_attn_c64_b16_traffic.md")
COPY_BYTES = 1 << 30  # copy-probe size: 1 GiB read + 1 GiB written, well above the 256 MB MALL
ATTN_KERNELS = ("attn_plan_kernel", "attn_bf16_kernel", "attn_merge_kernel")
ACCEPT_KERNELS = ("rowstats_kernel", "draw_kernel", "chunksum_kernel", "search_kernel")
# per call kind: its kernels, the kernel dispatched once per call, where the bench records
# the call's algorithmic bytes
TRAFFIC_CALLS = {
    "attention": (ATTN_KERNELS, "attn_bf16_kernel", ("roofline", "algorithmic_bytes")),
    "acceptance": (ACCEPT_KERNELS, "rowstats_kernel", ("kernels", "acceptance_algorithmic_bytes")),
}


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def attn_source_digest():
    import hashlib
    with open(ATTN_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def recorded_traffic(workload):
    """Bytes per call recorded for this workload and the current attention source, else None."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    fields = {}
    for line in open(TRAFFIC_FILE):
        line = line.strip().lstrip("-").strip()
        if ":" in line:
            k, v = line.split(":", 1)
            fields[k.strip()] = v.strip()
    if fields.get("workload") != workload or fields.get("attn_source_sha256") != attn_source_digest():
        return None
    try:
        return float(fields["traffic_bytes_per_call"])
    except (KeyError, ValueError):
        return None


def short_name(name):
    n = name.replace("void ", "").replace("sv::(anonymous namespace)::", "").replace("(anonymous namespace)::", "")
    depth = 0
    for i, ch in enumerate(n):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            n = n[:i]
            break
    return n if len(n) <= 90 else n[:87] + "..."


def summarize_trace(stats_csv):
    """Markdown table of a rocprofv3 --stats kernel summary (run_kernel_stats.csv)."""
    import csv
    rows = list(csv.DictReader(open(stats_csv)))
    out = ["| kernel | calls | avg us | min us | max us | share |", "|---|---|---|---|---|---|"]
    for r in rows:
        out.append(f"| `{short_name(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                   f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | {float(r['Percentage']):.1f}% |")
    run = [r for r in rows if "attn_bf16_kernel" in r["Name"] or "attn_merge_kernel" in r["Name"]]
    if run:
        # average kernel time of one attention run (the persistent kernel and the merge); the
        # plan is built by its own kernel only where a call builds it (sv_verify_attn)
        tot = sum(float(r["AverageNs"]) for r in run) / 1e3
        plan = [float(r["AverageNs"]) / 1e3 for r in rows if "attn_plan_kernel" in r["Name"]]
        out.append("")
        out.append(f"attention run per call (attention + merge kernels): {tot:.1f} us"
                   + (f"; plan kernel where a call builds its own plan: {plan[0]:.1f} us" if plan else ""))
    return "\n".join(out)


def summarize_traffic(fetch_dir, write_dir, call="attention"):
    """FETCH_SIZE / WRITE_SIZE per dispatch, scaled by the copy probe, as traffic per call
    of `call` (attention: sv_verify_attn; acceptance: sv_spec_accept)."""
    kernels, main_kernel, alg_key = TRAFFIC_CALLS[call]
    import csv
    import collections

    def per_kernel(d, counter):
        vals = collections.defaultdict(list)
        for r in csv.DictReader(open(os.path.join(d, "run_counter_collection.csv"))):
            if r["Counter_Name"] == counter:
                vals[r["Kernel_Name"]].append(float(r["Counter_Value"]))
        return vals

    fetch = per_kernel(fetch_dir, "FETCH_SIZE")
    write = per_kernel(write_dir, "WRITE_SIZE")

    def pick(vals, key):
        return {k: v for k, v in vals.items() if key in k}

    cf, cw = pick(fetch, "neg_kernel"), pick(write, "neg_kernel")
    assert cf and cw, "copy probe kernel not found in the counter runs"
    copy_fetch_kib = sum(sum(v) for v in cf.values()) / sum(len(v) for v in cf.values())
    copy_write_kib = sum(sum(v) for v in cw.values()) / sum(len(v) for v in cw.values())
    f_fetch = COPY_BYTES / (copy_fetch_kib * 1024)
    f_write = COPY_BYTES / (copy_write_kib * 1024)
    out = ["| kernel | dispatches | FETCH_SIZE KiB/dispatch | WRITE_SIZE KiB/dispatch |", "|---|---|---|---|"]
    for k in sorted(set(fetch) | set(write)):
        if not (any(a in k for a in kernels) or "neg_kernel" in k):
            continue
        fv, wv = fetch.get(k, [0.0]), write.get(k, [0.0])
        out.append(f"| `{short_name(k)}` | {len(fv)} | {sum(fv) / len(fv):.0f} | {sum(wv) / len(wv):.0f} |")
    main_calls = sum(len(v) for k, v in fetch.items() if main_kernel in k)
    tf = sum(sum(v) for k, v in fetch.items() if any(a in k for a in kernels)) / main_calls
    tw = sum(sum(v) for k, v in write.items() if any(a in k for a in kernels)) / main_calls
    traffic = tf * 1024 * f_fetch + tw * 1024 * f_write
    bench = {}
    bj = os.path.join(fetch_dir, "bench.json")
    if os.path.exists(bj):
        lines = [l for l in open(bj) if l.startswith("{")]
        if lines:
            bench = json.loads(lines[-1])
    alg = bench.get(alg_key[0], {}).get(alg_key[1])
    out += ["",
            f"- copy probe: {COPY_BYTES} bytes read and written; FETCH_SIZE {copy_fetch_kib:.0f} KiB, "
            f"WRITE_SIZE {copy_write_kib:.0f} KiB; scale factors fetch {f_fetch:.4f}, write {f_write:.4f}",
            f"- calls: {main_calls}",
            f"- fetch_bytes_per_call: {tf * 1024 * f_fetch:.0f}",
            f"- write_bytes_per_call: {tw * 1024 * f_write:.0f}",
            f"- traffic_bytes_per_call: {traffic:.0f}"]
    if alg:
        out.append(f"- algorithmic_bytes_per_call: {alg:.0f} (traffic / algorithmic = {traffic / alg:.3f})")
    out.append(f"- workload: {bench.get('config', {}).get('workload', '?').split(':')[0]}")
    if call == "attention":  # the digest of the source that ran (recorded by the bench run itself)
        out.append(f"- attn_source_sha256: {bench.get('roofline', {}).get('attn_source_sha256', '?')}")
    return "\n".join(out)


def copy_probe():
    """A plain elementwise copy (y = -x, fp32) of COPY_BYTES, three times: calibrates
    the FETCH_SIZE / WRITE_SIZE counters against a known byte count."""
    import torch
    src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda").uniform_()
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    del src, dst


# the paper's own figures are end-to-end serving numbers on other hardware: context only
PAPER_CONTEXT = ("AngelSpec reports no kernel timings; end to end, on 8x H20 (TP=8, vLLM, Hy3-295B-A21B), its "
                 "8-token block drafter serves 1.98-2.40x the tokens/s of plain decoding at concurrency 4-64, "
                 "and D-cut adds 3.0/9.2/15.7% on live traffic at concurrency 48/56/64")
READ_PROBE_BYTES = 2 << 30  # streaming-read probe: 2 GiB, eight times the last-level cache
WARM_SECONDS = 0.2  # untimed steps before a timed loop: at least the asked-for count and this long


def read_probe(steps=10):
    """Measured streaming-read bandwidth (GB/s) of a plain kernel (libsvprobe.so: one
    workgroup per 32 KB chunk, non-temporal 16-byte loads), the practical ceiling for
    the HBM-bound kernels; mean of `steps` back-to-back reads of READ_PROBE_BYTES."""
    import ctypes
    import torch
    from paper_2607_25852_amd import build
    lib = ctypes.CDLL(build.PROBE_LIB)
    lib.svprobe_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p]
    lib.svprobe_stream_read.restype = ctypes.c_int32
    buf = torch.empty(READ_PROBE_BYTES // 4, dtype=torch.float32, device="cuda").uniform_()
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()

    def once():
        st = lib.svprobe_stream_read(buf.data_ptr(), READ_PROBE_BYTES, sink.data_ptr(), stream.cuda_stream)
        if st != 0:
            raise RuntimeError(f"svprobe_stream_read failed: {st}")

    ms = time_loop(torch, stream, once, steps)
    del buf
    return READ_PROBE_BYTES / (ms * 1e-3) / 1e9


def attn_bytes(cfg, L, k):
    """Algorithmic HBM bytes of one verify-attention call: every visible K and V row
    read once per kv-head, plus q read and out written once."""
    import numpy as np
    e = 4 if cfg.dtype == "f32" else 2
    kv = float(np.sum(L + k)) * 2 * cfg.Hkv * cfg.d * e
    qo = float(np.sum(k)) * cfg.Hq * cfg.d * e * 2
    return kv + qo


def accept_bytes(cfg, k):
    """Algorithmic bytes of acceptance: each kept target row (n_i+1 per request) and
    each tested draft row (n_i) read once."""
    import numpy as np
    e = 4 if cfg.dtype == "f32" else 2
    n = k - 1
    return float(np.sum((n + 1) + n)) * cfg.V * e


def warm(torch, fn, min_calls, min_seconds):
    """Untimed calls of fn(): at least min_calls, and until min_seconds of them have run.
    The GPU's clocks drop within tens of milliseconds of idling and take about 20 ms of
    sustained work to come back (a round measured right after an idle gap is up to 20%
    slower), so every timed loop starts from a warm GPU, as in continuous serving."""
    calls = 0
    t0 = time.perf_counter()
    while calls < min_calls or time.perf_counter() - t0 < min_seconds:
        fn()
        calls += 1
        if calls % 8 == 0:  # keep the host at most a few calls ahead, so the time is the GPU's
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    return calls


def time_loop(torch, stream, fn, steps):
    """Mean milliseconds of fn() over `steps` back-to-back calls on `stream`, after warm-up
    calls (at least three, and at least 50 ms)."""
    warm(torch, fn, 3, 0.05)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(steps):
        fn()
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / steps


def workload_text(cfg):
    """One-line description of a workload from its configuration."""
    kind = cfg.kv[0]
    if kind == "lognormal":
        ctx = f"lognormal context median {cfg.kv[1]} in [{cfg.kv[3]}, {cfg.kv[4]}]"
    elif kind == "uniform":
        ctx = f"context uniform in [{cfg.kv[1]}, {cfg.kv[2]}]"
    else:
        ctx = "contexts " + "/".join(str(x) for x in cfg.kv[1:])
    budget = {"cost": "cost-table budget", "given": "verify depths k_i ~ U{1..b} given"}.get(
        cfg.budget[0], f"fixed budget K={cfg.budget[1] if len(cfg.budget) > 1 else '?'}")
    return (f"{cfg.name}: concurrency {cfg.R}, block {cfg.b}, Hq {cfg.Hq}/Hkv {cfg.Hkv}/d {cfg.d}, {ctx}, "
            f"page {cfg.page}, vocab {cfg.V}, {budget}")


def cpu_model():
    """The host CPU's model name as lscpu reports it (else /proc/cpuinfo)."""
    import subprocess
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def host_threads():
    """Host threads this process may use (its CPU affinity)."""
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def host_inputs(rnd, reqs):
    """Host copies of what the oracle needs for requests `reqs` of a device round: the
    queries of their kept rows, their page-table rows and the whole cache pool (copied back
    from the device, so that a round whose cache was drawn on the device can be timed on the
    host as well; the pool keeps its layout, so the sample walks the pages as the whole
    round would)."""
    import numpy as np
    import torch

    def host(t):
        if t.dtype == torch.bfloat16:
            return t.view(torch.int16).cpu().numpy().view(np.uint16)
        return t.cpu().numpy()

    qo = rnd.qo_host
    k = np.diff(qo)[reqs]
    qo_sub = np.zeros(len(reqs) + 1, np.int32)
    qo_sub[1:] = np.cumsum(k)
    q = np.ascontiguousarray(np.concatenate([rnd.kv["q_full"][i, :k[j]] for j, i in enumerate(reqs)]))
    if "k_cache" not in rnd.kv:
        rnd.kv["k_cache"], rnd.kv["v_cache"] = host(rnd.k_cache), host(rnd.v_cache)
    return dict(q=q, k_cache=rnd.kv["k_cache"], v_cache=rnd.kv["v_cache"],
                page_table=np.ascontiguousarray(rnd.kv["page_table"][reqs]), qo=qo_sub,
                kv_lens=(np.asarray(rnd.L)[reqs] + k).astype(np.int32))


def cpu_round(cfg, rnd, target_s, threads_all):
    """The oracle, as it stands, on a bounded sample of round `rnd`, per part, at one thread
    and at `threads_all` threads; each part's figure is the median of 3 repeats, scaled to the
    whole round by its share of the round's work.

    budget      the whole global selection (it is one decision over every request)
    attention   whole requests in a seeded random order (every row and head), as many as one
                single-thread repeat of about target_s holds, or the first rows of one request
                when a request alone takes much longer; scaled by the keys the sample reads
                against the keys the whole round reads
    acceptance  the first m requests, m sized the same way; scaled by the vocabulary rows
                read (n_i + 1 target rows and n_i draft rows per request)
    """
    import numpy as np
    import oracle
    from paper_2607_25852_amd import synth
    qo = rnd.qo_host
    k = np.diff(qo)
    R, b, Hq = cfg.R, cfg.b, cfg.Hq
    L = np.asarray(rnd.L, np.int64)
    mode = cfg.budget[0]
    cost = synth.profiled_cost(R, b) if mode == "cost" else None

    def budget():
        if mode == "cost":
            oracle.budget(rnd.lr["conf"], "cost", cost=cost)
        elif mode == "fixed":
            oracle.budget(rnd.lr["conf"], "fixed", fixed_budget=cfg.budget[1])

    # attention sample: whole requests (every row and head) in a seeded random order, as many
    # as one single-thread repeat of about target_s holds; if one request alone is much longer,
    # its first rows. Whole requests keep the cache reuse of the full batch (the rows of a
    # request walk the same keys one after another).
    keys_req = Hq * np.array([int(L[i]) * int(k[i]) + int(k[i]) * (int(k[i]) + 1) // 2 for i in range(R)],
                             np.float64)
    keys_round = float(keys_req.sum())
    order = np.random.default_rng(cfg.seed + 99).permutation(R)

    def attn_call(h, rows, heads):
        oracle.attention(h["q"], h["k_cache"], h["v_cache"], h["page_table"], h["qo"], h["kv_lens"],
                         dtype=cfg.dtype, units=(rows, heads))

    # acceptance sample: the first m requests
    tfull = rnd.lr["target_full"]
    dft = rnd.lr["draft"]

    def acc_inputs(m):
        qm = qo[:m + 1]
        return (synth.pack_rows(tfull[:m], qm), dft[:m], rnd.lr["draft_tokens"][:m], qm, rnd.ua_host[:m],
                rnd.us_host[:m])

    rows_req = (2 * k - 1).astype(np.float64)

    def acceptance(args_):
        oracle.accept(*args_, kind="logits", dtype=cfg.dtype)

    def timed(fn, reps=3):
        ts = []
        for _ in range(reps):
            t = time.perf_counter()
            fn()
            ts.append(time.perf_counter() - t)
        return float(np.median(ts))

    # size the samples at one thread
    oracle.set_num_threads(1)
    i0 = int(order[0])
    h0 = host_inputs(rnd, order[:1])
    t_row = timed(lambda: attn_call(h0, np.zeros(Hq, np.int32), np.arange(Hq, dtype=np.int32)), reps=1)
    per_key = t_row / (Hq * (float(L[i0]) + 1.0))
    if keys_req[i0] * per_key <= 2.0 * target_s:  # time the whole first request for a better rate
        nr0 = int(h0["qo"][-1])
        t0 = timed(lambda: attn_call(h0, np.repeat(np.arange(nr0, dtype=np.int32), Hq),
                                     np.tile(np.arange(Hq, dtype=np.int32), nr0)), reps=1)
        per_key = t0 / keys_req[i0]
    est = np.cumsum(keys_req[order]) * per_key
    if est[0] > 2.0 * target_s:
        h = h0
        keys_rows = Hq * (float(L[i0]) + np.arange(int(k[i0])) + 1.0)
        n = int(max(1, min(int(k[i0]), target_s // (per_key * keys_rows[0]))))
        units = (np.repeat(np.arange(n, dtype=np.int32), Hq), np.tile(np.arange(Hq, dtype=np.int32), n))
        keys_sample = float(keys_rows[:n].sum())
        what = f"the first {n} of {int(k[i0])} rows of one request (context {int(L[i0])}), every head"
    else:
        cnt = max(1, int(np.searchsorted(est, target_s, side="right")))
        reqs = np.sort(order[:cnt])
        h = host_inputs(rnd, reqs) if cnt > 1 else h0
        nr = int(h["qo"][-1])
        units = (np.repeat(np.arange(nr, dtype=np.int32), Hq), np.tile(np.arange(Hq, dtype=np.int32), nr))
        keys_sample = float(keys_req[reqs].sum())
        what = f"{cnt} of {R} whole requests (seeded random choice), every row and head"
    del h0

    def attention():
        attn_call(h, *units)

    m = 1
    while True:
        a_in = acc_inputs(m)
        t = timed(lambda: acceptance(a_in), reps=1)
        if t >= 0.5 * target_s or m == R:
            break
        m = min(R, max(m * 2, int(m * target_s / max(t, 1e-4))))
    acc_args = acc_inputs(m)
    scale_attn = keys_round / keys_sample
    scale_acc = float(rows_req.sum()) / float(rows_req[:m].sum())
    out = {}
    for th in (1, threads_all):
        oracle.set_num_threads(th)
        parts = {"budget": timed(budget) if mode != "given" else 0.0,
                 "attention": timed(attention) * scale_attn,
                 "acceptance": timed(lambda: acceptance(acc_args)) * scale_acc}
        tot = sum(parts.values())
        out[f"threads_{th}"] = {"threads": oracle.num_threads(), "round_seconds": tot,
                                "verified_drafts_per_s": float(np.sum(k - 1)) / tot,
                                "part_seconds": parts}
    oracle.set_num_threads(threads_all)
    out["sample"] = (f"budget: whole round; attention: {what} "
                     f"(x{scale_attn:.1f} by keys read); acceptance: first {m} of {R} requests "
                     f"(x{scale_acc:.2f} by rows read); median of 3 repeats per part")
    return out


def time_round(torch, rnds, steps, stream):
    """Wall-clock time per step over `steps` whole rounds (input copies in turn) with nothing
    else on the stream; then the same steps again with HIP events around each call.
    Returns (ms per step, {call: mean ms}); the calls are the round's own (DeviceRound.calls:
    prepare, attention, acceptance, or budget, pack, attention, acceptance)."""
    import numpy as np
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(steps):
        rnds[s % len(rnds)].run()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    names = [c for c, _ in rnds[0].calls()]
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)] for _ in range(steps)]
    torch.cuda.synchronize()
    for s in range(steps):
        e, r = ev[s], rnds[s % len(rnds)]
        e[0].record(stream)
        for j, (_, fn) in enumerate(r.calls()):
            fn()
            e[j + 1].record(stream)
    torch.cuda.synchronize()
    per = {c: float(np.mean([e[j].elapsed_time(e[j + 1]) for e in ev])) for j, c in enumerate(names)}
    return ms, per


def call_figures(per):
    """The per-call times of time_round as the JSON line's `kernels` entries (us)."""
    out = {f"{c}_us": v * 1e3 for c, v in per.items()}
    for c in ("prepare", "budget", "pack"):
        out.setdefault(f"{c}_us", None)
    return out


def copies_for(cfg, L, k, floor_bytes=768 << 20, lo=3, hi=16):
    """Input copies used in turn: enough that the bytes one pass over them reads are at least
    three times the 256 MB last-level cache."""
    import math
    per = attn_bytes(cfg, L, k) + accept_bytes(cfg, k)
    return max(lo, min(hi, math.ceil(floor_bytes / per)))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="c64_b16")
    ap.add_argument("--kv-split", type=int, default=0)
    ap.add_argument("--rotate", type=int, default=3,
                    help="copies of the round's inputs used in turn, so that every step reads from HBM rather "
                         "than the 256 MB last-level cache")
    ap.add_argument("--range", default="all",
                    help="other workloads timed after the main one and reported under 'workloads' "
                         "(comma-separated names, 'all' or 'none')")
    ap.add_argument("--cpu-seconds", type=float, default=1.0,
                    help="single-thread host time of one sampled repeat of each part of the oracle baseline "
                         "(0: skip the baseline)")
    ap.add_argument("--copy-probe", action="store_true", help="also run a 1 GiB copy kernel (counter calibration)")
    ap.add_argument("--summarize-trace", metavar="CSV", help="print a rocprofv3 kernel-stats CSV as markdown")
    ap.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print HBM traffic per call from two rocprofv3 --pmc runs")
    ap.add_argument("--traffic-call", choices=sorted(TRAFFIC_CALLS), default="attention",
                    help="the call --summarize-traffic reports")
    ap.add_argument("--unfused", action="store_true",
                    help="step as separate calls: sv_alloc_budget, sv_pack_verify, sv_verify_attn (its own plan), "
                         "sv_spec_accept")
    ap.add_argument("--step-only", action="store_true",
                    help="time the steps only: no greedy, packing, draft-statistics, graph, read-probe, other "
                         "workloads or host baseline (for counter runs)")
    args = ap.parse_args()
    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace))
        return
    if args.summarize_traffic:
        print(summarize_traffic(*args.summarize_traffic, call=args.traffic_call))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the round's kernels run on a single MI355X and the library "
              "has no multi-GPU path; run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2607_25852_amd import binding, synth
    from paper_2607_25852_amd.round import DeviceRound, to_dev

    binding.load()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    cfg = synth.CONFIGS[args.workload]
    log("generating inputs", cfg.name)
    t0 = time.perf_counter()
    rnd = DeviceRound(cfg, kind="logits", kv_split=args.kv_split, fused=not args.unfused)
    rnds = [rnd] + [rnd.replica() for _ in range(max(1, args.rotate) - 1)]
    torch.cuda.synchronize()
    log(f"inputs resident ({time.perf_counter() - t0:.1f} s, {len(rnds)} copies); K={rnd.K}")
    k = np.diff(rnd.qo_host)
    drafts = int(np.sum(k - 1))

    stream = torch.cuda.current_stream()
    turn = [0]

    def step():
        rnds[turn[0] % len(rnds)].run()
        turn[0] += 1

    for r in rnds:
        r.run()
    torch.cuda.synchronize()
    # the selection is deterministic: the timed steps see the same qo_indptr in every copy
    for r in rnds:
        assert np.array_equal(r.qo.cpu().numpy(), rnd.qo_host)
    committed = int(np.sum(rnd.accept_len.cpu().numpy() + 1))
    n_warm = warm(torch, step, args.warmup, WARM_SECONDS)

    # the timed steps: the calls of a round back to back, nothing else on the stream (HIP
    # events between the calls would add about 10 us per step of their own); then the same
    # steps with events around each call
    ms_step, per = time_round(torch, rnds, args.steps, stream)
    t_attn, t_acc = per["attention"], per["acceptance"]
    value = drafts / (ms_step * 1e-3)
    a_bytes = attn_bytes(cfg, rnd.L, k)
    x_bytes = accept_bytes(cfg, k)
    a_gbs = a_bytes / (t_attn * 1e-3) / 1e9
    x_gbs = x_bytes / (t_acc * 1e-3) / 1e9
    log(f"step {ms_step:.3f} ms: " + ", ".join(f"{c} {v * 1e3:.1f} us" for c, v in per.items())
        + f" (attention {a_gbs:.0f} GB/s, acceptance {x_gbs:.0f} GB/s)")

    def post_step_figures():
        """Figures of the calls outside the step, on the same round (first input copy)."""
        # greedy verification (temperature 0) on the same round, outside the timed steps: the
        # argmax pass reads only the kept target rows
        gdesc = binding.accept_desc(cfg.R, cfg.b, cfg.V, binding.SV_LOGITS,
                                    binding.SV_F32 if cfg.dtype == "f32" else binding.SV_BF16, 0.0)
        gws = torch.empty(max(binding.accept_workspace_size(gdesc), 256), dtype=torch.uint8, device="cuda")

        def greedy():
            binding.spec_accept(gdesc, rnd.target, None, rnd.tokens, rnd.qo, None, None, rnd.accept_len,
                                rnd.out_tokens, rnd.flags, gws)

        t_greedy = time_loop(torch, stream, greedy, args.steps)
        g_bytes = float(rnd.K) * cfg.V * (4 if cfg.dtype == "f32" else 2)

        # the KV append of the same round, outside the timed steps; it writes the kept
        # positions' own keys and values (gathered from the cache) back to their slots, so the
        # round's cache is unchanged
        e_sz = 4 if cfg.dtype == "f32" else 2
        pt_h = rnd.kv["page_table"]
        k_new_h = np.empty((rnd.K, cfg.Hkv, cfg.d), rnd.kv["k_cache"].dtype)
        v_new_h = np.empty_like(k_new_h)
        for i in range(cfg.R):
            for j in range(int(k[i])):
                s_ = int(rnd.L[i]) + j
                k_new_h[rnd.qo_host[i] + j] = rnd.kv["k_cache"][pt_h[i, s_ // cfg.page], :, s_ % cfg.page]
                v_new_h[rnd.qo_host[i] + j] = rnd.kv["v_cache"][pt_h[i, s_ // cfg.page], :, s_ % cfg.page]
        k_new, v_new = to_dev(k_new_h), to_dev(v_new_h)
        apdesc = binding.append_desc(cfg.R, rnd.K, cfg.b, cfg.Hkv, cfg.d, cfg.page, pt_h.shape[1], rnd.kv["num_pages"],
                                     binding.SV_F32 if cfg.dtype == "f32" else binding.SV_BF16)

        def append():
            binding.append_kv(apdesc, k_new, v_new, rnd.page_table, rnd.qo, rnd.ctx_lens, rnd.k_cache, rnd.v_cache)

        t_pack_alone = time_loop(torch, stream, rnd.run_pack, args.steps)
        # the round's set-up and attention as separate calls (sv_alloc_budget alone;
        # sv_verify_attn building its own work plan), for comparison with the fused step
        t_budget_alone = time_loop(torch, stream, rnd.run_budget, args.steps) if rnd.mode != "given" else None
        t_attn_full = time_loop(torch, stream, rnd.run_attn, args.steps)
        t_append = time_loop(torch, stream, append, args.steps)
        ap_bytes = 4.0 * rnd.K * cfg.Hkv * cfg.d * e_sz

        # the drafter's side: softmax statistics and confidences of every draft row, then the
        # acceptance that takes the draft rows' statistics instead of re-reading them (same
        # outputs bit for bit), both on the same round and outside the timed steps
        dsdesc = binding.draft_stats_desc(cfg.R, cfg.b - 1, cfg.V, binding.SV_F32 if cfg.dtype == "f32" else binding.SV_BF16)
        ds_ws = torch.empty(max(binding.draft_stats_workspace_size(dsdesc), 256), dtype=torch.uint8, device="cuda")
        ds_stats = torch.empty((cfg.R * (cfg.b - 1), 2), dtype=torch.float32, device="cuda")
        ds_conf = torch.empty(cfg.R * (cfg.b - 1), dtype=torch.float32, device="cuda")

        def dstats():
            binding.draft_stats(dsdesc, rnd.draft, ds_stats, ds_conf, ds_ws)

        def accept_with_stats():
            binding.spec_accept_stats(rnd.xdesc, rnd.target, rnd.draft, ds_stats, rnd.tokens, rnd.qo, rnd.u_accept,
                                      rnd.u_sample, rnd.accept_len, rnd.out_tokens, rnd.flags, rnd.acc_ws)

        t_dstats = time_loop(torch, stream, dstats, args.steps)
        ds_bytes = float(cfg.R * (cfg.b - 1)) * cfg.V * e_sz
        rnd.run_accept()
        ref_out = (rnd.accept_len.clone(), rnd.out_tokens.clone())
        t_acc_stats = time_loop(torch, stream, accept_with_stats, args.steps)
        assert torch.equal(rnd.accept_len, ref_out[0]) and torch.equal(rnd.out_tokens, ref_out[1])
        xs_bytes = float(rnd.K) * cfg.V * e_sz

        # the round captured as HIP graphs: one graph per input copy, replayed in turn (the
        # eager step's access pattern), and one graph holding a round on every copy back to
        # back. Launch shapes do not depend on the budget's choice, so one graph serves every
        # round of a shape.
        gs = torch.cuda.Stream()
        gs.wait_stream(stream)
        with torch.cuda.stream(gs):
            for r in rnds:
                r.run()
        stream.wait_stream(gs)
        torch.cuda.synchronize()
        graphs = []
        for r in rnds:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                r.run()
            graphs.append(g)
        chain = torch.cuda.CUDAGraph()
        with torch.cuda.graph(chain):
            for r in rnds:
                r.run()
        torch.cuda.synchronize()
        turn = [0]

        def replay():
            graphs[turn[0] % len(graphs)].replay()
            turn[0] += 1

        def eager():
            rnds[turn[0] % len(rnds)].run()
            turn[0] += 1

        def chained():
            chain.replay()

        # eager steps and both graph forms, in alternating blocks (clock and neighbour drift hit
        # all three alike); medians over the blocks
        blocks = {"eager": [], "graph": [], "chain": []}
        for _ in range(3):
            blocks["eager"].append(time_loop(torch, stream, eager, args.steps))
            blocks["graph"].append(time_loop(torch, stream, replay, args.steps))
            blocks["chain"].append(time_loop(torch, stream, chained, max(1, args.steps // len(rnds))) / len(rnds))
        t_eager, t_graph, t_chain = (float(np.median(blocks[key])) for key in ("eager", "graph", "chain"))
        del graphs, chain

        return {"greedy_acceptance_us": t_greedy * 1e3,
                "greedy_acceptance_gbs": g_bytes / (t_greedy * 1e-3) / 1e9,
                "greedy_acceptance_algorithmic_bytes": g_bytes,
                "pack_alone_us": t_pack_alone * 1e3, "append_us": t_append * 1e3,
                "budget_alone_us": None if t_budget_alone is None else t_budget_alone * 1e3,
                "attention_with_own_plan_us": t_attn_full * 1e3,
                "append_gbs": ap_bytes / (t_append * 1e-3) / 1e9, "append_algorithmic_bytes": ap_bytes,
                "draft_stats_us": t_dstats * 1e3, "draft_stats_gbs": ds_bytes / (t_dstats * 1e-3) / 1e9,
                "draft_stats_algorithmic_bytes": ds_bytes,
                "acceptance_with_draft_stats_us": t_acc_stats * 1e3,
                "acceptance_with_draft_stats_gbs": xs_bytes / (t_acc_stats * 1e-3) / 1e9,
                "acceptance_with_draft_stats_algorithmic_bytes": xs_bytes,
                "graph_step_us": t_graph * 1e3, "graph_chain_step_us": t_chain * 1e3,
                "graph_chain_rounds": len(rnds), "eager_step_us_event_timed": t_eager * 1e3}

    extra = {} if args.step_only else post_step_figures()
    read_gbs = None
    if not args.step_only:
        read_gbs = read_probe()
        log(f"streaming-read probe: {read_gbs:.0f} GB/s")
    if args.copy_probe:
        log("copy probe")
        copy_probe()
    traffic = recorded_traffic(cfg.name) if args.kv_split == 0 else None

    threads_all = host_threads()
    cpu = None
    if args.cpu_seconds > 0 and not args.step_only:
        log(f"timing the oracle on the host ({cfg.name})")
        cr = cpu_round(cfg, rnd, args.cpu_seconds, threads_all)
        ta = cr[f"threads_{threads_all}"]
        cpu = dict(value=ta["verified_drafts_per_s"], unit="verified draft tokens/s", cores=ta["threads"],
                   kind="oracle", sample=cr["sample"], cpu_model=cpu_model(),
                   single_thread_value=cr["threads_1"]["verified_drafts_per_s"],
                   part_seconds=ta["part_seconds"], part_seconds_single_thread=cr["threads_1"]["part_seconds"],
                   workloads={})
    main_round_bytes = sum(r.device_bytes() for r in rnds)
    del rnds
    torch.cuda.empty_cache()

    # the other workloads: each timed like the main one (fresh inputs, copies in turn), its
    # cache drawn on the device; then its host baseline on a sample of the same round
    names = [] if args.step_only or args.range == "none" else (
        [n for n in synth.CONFIGS if n != cfg.name] if args.range == "all" else args.range.split(","))
    ranges = {}
    for name in names:
        c2 = synth.CONFIGS[name]
        t1 = time.perf_counter()
        r0 = DeviceRound(c2, kind="logits", kv="device", fused=not args.unfused)
        k2 = np.diff(r0.qo_host)
        n_copies = copies_for(c2, r0.L, k2)
        rr = [r0] + [r0.replica() for _ in range(n_copies - 1)]
        turn2 = [0]

        def step2():
            rr[turn2[0] % len(rr)].run()
            turn2[0] += 1

        warm(torch, step2, args.warmup, WARM_SECONDS)
        ms2, per2 = time_round(torch, rr, args.steps, stream)
        d2 = int(np.sum(k2 - 1))
        ab2, xb2 = attn_bytes(c2, r0.L, k2), accept_bytes(c2, k2)
        fig = {"workload": workload_text(c2), "concurrency": c2.R, "block": c2.b, "verified_positions": int(r0.K),
               "verified_drafts": d2, "budget_ratio_index": None if r0.mode == "given" else int(r0.sel[1].item()),
               "input_copies": n_copies, "step_us": ms2 * 1e3, "verified_drafts_per_s": d2 / (ms2 * 1e-3),
               **call_figures(per2),
               "attention_frac": ab2 / (per2["attention"] * 1e-3) / 1e9 / HBM_PEAK_GBS,
               "acceptance_frac": xb2 / (per2["acceptance"] * 1e-3) / 1e9 / HBM_PEAK_GBS,
               "attention_algorithmic_bytes": ab2, "acceptance_algorithmic_bytes": xb2}
        ranges[name] = fig
        log(f"{name}: step {ms2 * 1e3:.1f} us, {fig['verified_drafts_per_s']:.3g} drafts/s, attention "
            f"{fig['attention_frac']:.3f}, acceptance {fig['acceptance_frac']:.3f} ({n_copies} copies, "
            f"{time.perf_counter() - t1:.1f} s)")
        if cpu is not None:
            cr = cpu_round(c2, r0, args.cpu_seconds, threads_all)
            cpu["workloads"][name] = cr
            log(f"{name}: oracle {cr['threads_1']['round_seconds']:.2f} s per round at 1 thread, "
                f"{cr[f'threads_{threads_all}']['round_seconds']:.2f} s at {threads_all}")
        del rr, r0
        torch.cuda.empty_cache()

    res = {
        "metric": "verified draft tokens/sec/GPU",
        "value": value,
        "unit": "verified draft tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_steps_run": n_warm,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": workload_text(cfg),
                   "concurrency": cfg.R, "block": cfg.b, "verified_positions": int(rnd.K),
                   "verified_drafts": drafts,
                   "budget_ratio_index": None if rnd.mode == "given" else int(rnd.sel[1].item()),
                   "input_copies": max(1, args.rotate), "input_bytes": main_round_bytes,
                   "parallelism": "single GPU"},
        "roofline": {"bound": "hbm",
                     "kernel": ("sv_verify_attn_run (split-KV attention + partial merge; the work plan is built "
                                "once per round by sv_prepare_round)" if rnd.fused and rnd.mode != "given" else
                                "sv_verify_attn (plan + split-KV attention + partial merge)"),
                     "achieved": a_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": a_gbs / HBM_PEAK_GBS,
                     "traffic": traffic, "traffic_unit": "HBM bytes per call", "algorithmic_bytes": a_bytes,
                     "call_us": t_attn * 1e3, "attn_source_sha256": attn_source_digest(),
                     "measured_read_peak": read_gbs,
                     "frac_of_measured_read_peak": a_gbs / read_gbs if read_gbs else None},
        "kernels": {**call_figures(per),
                    "acceptance_gbs": x_gbs, "acceptance_frac": x_gbs / HBM_PEAK_GBS,
                    "acceptance_algorithmic_bytes": x_bytes,
                    **extra},
        "verified_positions_per_s": rnd.K / (ms_step * 1e-3),
        "committed_tokens_per_s": committed / (ms_step * 1e-3),
        "workloads": ranges,
        "cpu_baseline": cpu,
        "paper_context": PAPER_CONTEXT,
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
