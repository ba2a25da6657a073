"""Benchmark of one draft-verify round on one MI355X.

A step is the whole round on resident inputs, on one stream:
  sv_alloc_budget (D-cut: prefix scores, global top-K, cost-table ratio, packing)
  sv_verify_attn  (one layer of verify attention over the paged KV cache)
  sv_spec_accept  (softmax of bf16 logits, accept test, first-reject cut, residual/bonus draw)
Workload (default): concurrency 64, block 16 (15 drafts + the certain token), bf16,
64 query / 8 KV heads of dim 128, committed context lognormal (median 4096, clipped
to [512, 32768]) in 64-token pages, vocabulary 131072, per-request draft noise drawn
from {0.3, 1.0, 2.0}, budget ratio chosen by a linear-plus-step cost table.

Metric: verified draft tokens per second (sum of kept drafts n_i per step / step time).
One JSON line on stdout; progress on stderr.
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
ACCEPT_KERNELS = ("rowstats_kernel", "chunksum_kernel", "search_kernel")
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
    attn = [r for r in rows if any(k in r["Name"] for k in ATTN_KERNELS)]
    if attn:
        calls = max(int(r["Calls"]) for r in attn if "attn_bf16_kernel" in r["Name"]) if any(
            "attn_bf16_kernel" in r["Name"] for r in attn) else 1
        tot = sum(float(r["TotalDurationNs"]) for r in attn) / calls / 1e3
        out.append("")
        out.append(f"sv_verify_attn kernels per call (plan + attention + merge): {tot:.1f} us")
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


def time_loop(torch, stream, fn, steps):
    """Mean milliseconds of fn() over `steps` back-to-back calls on `stream`, after three
    untimed calls."""
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
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
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, rnd, min_seconds):
    """The oracle, as it stands, on the same round: the budget over the whole batch (as
    the workload defines it), then attention (every row and head) and acceptance of every
    request; repeated until at least min_seconds of host time have passed. Also the mean
    host time of each part."""
    import numpy as np
    import oracle
    from paper_2607_25852_amd import synth
    qo = rnd.qo_host
    k = np.diff(qo)
    kv = rnd.kv
    q = synth.pack_rows(kv["q_full"], qo)
    target = synth.pack_rows(rnd.lr["target_full"], qo)
    mode = cfg.budget[0]
    cost = synth.profiled_cost(cfg.R, cfg.b) if mode == "cost" else None
    parts = dict(budget=0.0, attention=0.0, acceptance=0.0)
    reps = 0
    t0 = time.perf_counter()
    while True:
        ta = time.perf_counter()
        if mode == "cost":
            oracle.budget(rnd.lr["conf"], "cost", cost=cost)
        elif mode == "fixed":
            oracle.budget(rnd.lr["conf"], "fixed", fixed_budget=cfg.budget[1])
        tb = time.perf_counter()
        oracle.attention(q, kv["k_cache"], kv["v_cache"], kv["page_table"], qo, rnd.kv_lens_host, dtype=cfg.dtype)
        tc = time.perf_counter()
        oracle.accept(target, rnd.lr["draft"], rnd.lr["draft_tokens"], qo, rnd.ua_host, rnd.us_host,
                      kind="logits", dtype=cfg.dtype)
        td = time.perf_counter()
        parts["budget"] += tb - ta
        parts["attention"] += tc - tb
        parts["acceptance"] += td - tc
        reps += 1
        dt = td - t0
        if dt >= min_seconds:
            break
    drafts = float(np.sum(k - 1)) * reps
    return dict(value=drafts / dt, unit="verified draft tokens/s", cores=oracle.num_threads(), kind="oracle",
                sample=f"the whole round ({cfg.R} requests, {int(np.sum(k - 1))} kept drafts: budget, attention "
                       f"of every row and head, acceptance) repeated {reps}x in {dt:.1f} s",
                cpu_model=cpu_model(), part_seconds={kk: v / reps for kk, v in parts.items()})


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
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="host time for the oracle baseline (0: skip)")
    ap.add_argument("--copy-probe", action="store_true", help="also run a 1 GiB copy kernel (counter calibration)")
    ap.add_argument("--summarize-trace", metavar="CSV", help="print a rocprofv3 kernel-stats CSV as markdown")
    ap.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print HBM traffic per call from two rocprofv3 --pmc runs")
    ap.add_argument("--traffic-call", choices=sorted(TRAFFIC_CALLS), default="attention",
                    help="the call --summarize-traffic reports")
    ap.add_argument("--step-only", action="store_true",
                    help="time the steps only: no greedy, packing, draft-statistics, graph or read-probe figures "
                         "(for counter runs)")
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
    rnds = [DeviceRound(cfg, kind="logits", kv_split=args.kv_split) for _ in range(max(1, args.rotate))]
    rnd = rnds[0]
    torch.cuda.synchronize()
    log(f"inputs resident ({time.perf_counter() - t0:.1f} s, {len(rnds)} copies); K={rnd.K}")
    k = np.diff(rnd.qo_host)
    drafts = int(np.sum(k - 1))

    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        for r in rnds:
            r.run()
    torch.cuda.synchronize()
    # the selection is deterministic: the timed steps see the same qo_indptr in every copy
    for r in rnds:
        assert np.array_equal(r.qo.cpu().numpy(), rnd.qo_host)
    committed = int(np.sum(rnd.accept_len.cpu().numpy() + 1))

    # the timed steps: the three calls back to back, nothing else on the stream (HIP events
    # between the calls would add about 10 us per step of their own)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for s in range(args.steps):
        r = rnds[s % len(rnds)]
        r.run_budget()
        r.run_attn()
        r.run_accept()
    torch.cuda.synchronize()
    t_end = time.perf_counter()
    ms_step = (t_end - t_start) * 1e3 / args.steps
    # per-call times: the same steps again, with HIP events around each call
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    for s in range(args.steps):
        e, r = ev[s], rnds[s % len(rnds)]
        e[0].record(stream)
        r.run_budget()
        e[1].record(stream)
        r.run_attn()
        e[2].record(stream)
        r.run_accept()
        e[3].record(stream)
    torch.cuda.synchronize()
    t_budget = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    t_attn = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    t_acc = float(np.mean([e[2].elapsed_time(e[3]) for e in ev]))
    value = drafts / (ms_step * 1e-3)
    a_bytes = attn_bytes(cfg, rnd.L, k)
    x_bytes = accept_bytes(cfg, k)
    a_gbs = a_bytes / (t_attn * 1e-3) / 1e9
    x_gbs = x_bytes / (t_acc * 1e-3) / 1e9
    log(f"step {ms_step:.3f} ms: budget {'given depths' if rnd.mode == 'given' else f'{t_budget * 1e3:.1f} us'}, "
        f"attention {t_attn * 1e3:.1f} us "
        f"({a_gbs:.0f} GB/s), acceptance {t_acc * 1e3:.1f} us ({x_gbs:.0f} GB/s)")

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

        # packing of the verify batch and the KV append of the same round, outside the timed
        # steps; the append writes the kept positions' own keys and values (gathered from the
        # cache) back to their slots, so the round's cache is unchanged
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
        ctx = to_dev(np.asarray(rnd.L, np.int32))
        blk_tok = to_dev(np.random.default_rng(cfg.seed).integers(0, cfg.V, size=(cfg.R, cfg.b)).astype(np.int32))
        p_tok = torch.empty(cfg.R * cfg.b, dtype=torch.int32, device="cuda")
        p_pos = torch.empty_like(p_tok)
        p_kvl = torch.empty(cfg.R, dtype=torch.int32, device="cuda")
        pdesc = binding.pack_desc(cfg.R, cfg.b, cfg.R * cfg.b)
        apdesc = binding.append_desc(cfg.R, rnd.K, cfg.b, cfg.Hkv, cfg.d, cfg.page, pt_h.shape[1], rnd.kv["num_pages"],
                                     binding.SV_F32 if cfg.dtype == "f32" else binding.SV_BF16)

        def pack():
            binding.pack_verify(pdesc, blk_tok, ctx, rnd.qo, p_tok, p_pos, p_kvl)

        def append():
            binding.append_kv(apdesc, k_new, v_new, rnd.page_table, rnd.qo, ctx, rnd.k_cache, rnd.v_cache)

        t_pack = time_loop(torch, stream, pack, args.steps)
        t_append = time_loop(torch, stream, append, args.steps)
        assert np.array_equal(p_kvl.cpu().numpy(), rnd.kv_lens_host)
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

        # the same round captured once as a HIP graph and replayed: the launch shapes do not
        # depend on the budget's choice, so one graph serves every round of this shape
        gs = torch.cuda.Stream()
        gs.wait_stream(stream)
        with torch.cuda.stream(gs):
            rnd.run()
        stream.wait_stream(gs)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            rnd.run()
        torch.cuda.synchronize()
        t_graph = time_loop(torch, stream, graph.replay, args.steps)

        return {"greedy_acceptance_us": t_greedy * 1e3,
                "greedy_acceptance_gbs": g_bytes / (t_greedy * 1e-3) / 1e9,
                "greedy_acceptance_algorithmic_bytes": g_bytes,
                "pack_us": t_pack * 1e3, "append_us": t_append * 1e3,
                "append_gbs": ap_bytes / (t_append * 1e-3) / 1e9, "append_algorithmic_bytes": ap_bytes,
                "draft_stats_us": t_dstats * 1e3, "draft_stats_gbs": ds_bytes / (t_dstats * 1e-3) / 1e9,
                "draft_stats_algorithmic_bytes": ds_bytes,
                "acceptance_with_draft_stats_us": t_acc_stats * 1e3,
                "acceptance_with_draft_stats_gbs": xs_bytes / (t_acc_stats * 1e-3) / 1e9,
                "acceptance_with_draft_stats_algorithmic_bytes": xs_bytes,
                "graph_step_us": t_graph * 1e3}

    extra = {} if args.step_only else post_step_figures()
    read_gbs = None
    if not args.step_only:
        read_gbs = read_probe()
        log(f"streaming-read probe: {read_gbs:.0f} GB/s")
    if args.copy_probe:
        log("copy probe")
        copy_probe()
    traffic = recorded_traffic(cfg.name) if args.kv_split == 0 else None

    cpu = None
    if args.cpu_seconds > 0:
        log("timing the oracle on the host")
        cpu = cpu_baseline(cfg, rnd, args.cpu_seconds)

    res = {
        "metric": "verified draft tokens/sec/GPU",
        "value": value,
        "unit": "verified draft tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
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
                   "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "kernel": "sv_verify_attn (plan + split-KV attention + partial merge)",
                     "achieved": a_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": a_gbs / HBM_PEAK_GBS,
                     "traffic": traffic, "traffic_unit": "HBM bytes per call", "algorithmic_bytes": a_bytes,
                     "call_us": t_attn * 1e3, "attn_source_sha256": attn_source_digest(),
                     "measured_read_peak": read_gbs,
                     "frac_of_measured_read_peak": a_gbs / read_gbs if read_gbs else None},
        "kernels": {"budget_us": None if rnd.mode == "given" else t_budget * 1e3,
                    "attention_us": t_attn * 1e3, "acceptance_us": t_acc * 1e3,
                    "acceptance_gbs": x_gbs, "acceptance_frac": x_gbs / HBM_PEAK_GBS,
                    "acceptance_algorithmic_bytes": x_bytes,
                    **extra},
        "verified_positions_per_s": rnd.K / (ms_step * 1e-3),
        "committed_tokens_per_s": committed / (ms_step * 1e-3),
        "cpu_baseline": cpu,
        "paper_context": PAPER_CONTEXT,
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
