"""Benchmark of the RPD commit step on one MI355X.

One step = one call of the whole commit step (masked-position compaction,
logit-lens projection with fused softmax statistics, cross-tile reduction
and stability scoring, budgeted commitment) on a seeded synthetic batch that
is resident in HBM before timing starts. Prints ONE JSON line on stdout;
progress goes to stderr.

Default workload: late decoding at the LLaDA-8B shape (d=4096, V=126464,
bf16, one 256-position canvas with 8 masked positions, the final K=4
layers), the regime where streaming the 1.04 GB unembedding bounds the step.
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 matrix peak
RIDGE_ROWS = 315             # projected rows where the projection turns compute-bound

METRIC = "masked positions scored+committed/sec at LLaDA-8B shape; MFMA % / HBM GB/s"
# What the paper reports about the cost of this step, for context only (another GPU, whole decodes with
# the backbone; nothing comparable to the step's own throughput here).
PAPER_CONTEXT = {
    "hardware": "one NVIDIA A6000, bf16, batch 1, 256-token canvas (Section 4.1)",
    "commit_step_time": None,
    "note": "the paper gives no absolute time for the projection, scoring and commitment; whole-decode "
            "runtime relative to Fast-dLLM is 1.03x for RPD and 0.96x for RPD-block, the backbone forward "
            "taking most of it (Section 4, decoding behavior and overhead, Figure 5c)",
}
CSRC = os.path.join(ROOT, "paper_2609_36452_amd", "csrc")
# the source files that define each projection variant's kernel
VARIANT_SOURCES = {v: ["rpd_device.h", "proj_stream.hip"] for v in
                   ("bf16_s32", "bf16_s64")}
VARIANT_SOURCES.update({v: ["rpd_device.h", "proj_big.hip"] for v in ("bf16_big", "bf16_big192", "bf16_big128")})
VARIANT_SOURCES["f32"] = ["rpd_device.h", "proj_f32.hip"]
VARIANT_KERNEL = {v: "k_proj_bf16_stream" for v in ("bf16_s32", "bf16_s64")}
VARIANT_KERNEL.update({v: "k_proj_bf16_big" for v in ("bf16_big", "bf16_big192", "bf16_big128")})
VARIANT_KERNEL["f32"] = "k_proj_f32"
COPY_PROBE_BYTES = 1 << 30     # fp32 elements read (and as many written) by the copy probe


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def code_tokens(src: str) -> str:
    """C++ source without its comments, whitespace runs collapsed to one
    space: what a counter measurement depends on (string and character
    literals are kept whole)."""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        elif c in "\"'":
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_source_sha(variant: str) -> str:
    """Hash of the code (comments and layout excluded) of the files that
    define a projection variant's kernel."""
    h = hashlib.sha256()
    for f in VARIANT_SOURCES[variant]:
        h.update(code_tokens(open(os.path.join(CSRC, f), encoding="utf-8").read()).encode())
        h.update(b"\0")
    return h.hexdigest()[:16]


def traffic_path(variant: str, workload: str) -> str:
    return os.path.join(ROOT, "profiles", f"proj_{variant}_{workload}_traffic.txt")


def read_traffic(variant: str, workload: str):
    """HBM bytes per projection launch from the committed rocprofv3 counter
    summary of this workload, if it was taken on the current source of the
    kernel; else None."""
    path = traffic_path(variant, workload)
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if "=" in line and not line.lstrip().startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha") != kernel_source_sha(variant):
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def copy_probe(torch) -> float:
    """A plain streaming copy of known size (read COPY_PROBE_BYTES, write as
    many) for scaling the HBM byte counters: three timed launches of torch.neg
    on fp32 buffers far larger than the last-level cache (after one that
    loads the kernel). Returns the copy's
    HBM rate in GB/s (bytes read + written over the average launch), a
    reference for what this particular GPU streams."""
    n = COPY_PROBE_BYTES // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.neg(src, out=dst)        # the first launch loads the kernel
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(3):
        torch.neg(src, out=dst)
    b.record()
    torch.cuda.synchronize()
    gbs = 2 * COPY_PROBE_BYTES * 3 / (a.elapsed_time(b) / 1e3) / 1e9
    log(f"copy probe: 3 launches, each reads {COPY_PROBE_BYTES} B and writes {COPY_PROBE_BYTES} B; {gbs:.0f} GB/s")
    del src, dst
    return gbs


def cpu_model() -> str:
    """The host CPU's model name (for the CPU baseline's context)."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def blas_threads() -> int:
    try:
        from threadpoolctl import threadpool_info
        n = [i["num_threads"] for i in threadpool_info() if i.get("user_api") == "blas"]
        if n:
            return int(max(n))
    except Exception:
        pass
    return os.cpu_count() or 1


def cpu_baseline(w, P, budget_s: float) -> dict:
    """The fp64 oracle, as it is, on the host cores over a bounded sample of
    the same workload: whole calls of the step while they fit the budget,
    else a prefix of its masked positions."""
    import numpy as np
    import oracle as O
    pos_all = O.masked_positions(w.mask)
    t0 = time.perf_counter()
    pos, layer = O.layer_stats_masked(w.hidden, w.w_u, w.mask, w.cfg.dtype)
    O.assemble(w.mask, pos, layer, P)
    t = time.perf_counter() - t0
    reps = 1
    while t * (reps + 1) / reps < budget_s and reps < 256:
        t0 = time.perf_counter()
        pos, layer = O.layer_stats_masked(w.hidden, w.w_u, w.mask, w.cfg.dtype)
        O.assemble(w.mask, pos, layer, P)
        t += time.perf_counter() - t0
        reps += 1
    n = len(pos_all)
    return {"value": n * reps / t, "unit": "positions/s", "cores": blas_threads(), "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"{reps} whole call(s) of the step ({n} masked positions x {w.cfg.K} layers, "
                      f"V={w.cfg.V}, d={w.cfg.d}) in float64, {t:.1f} s"}


def cpu_baseline_sampled(w, P, n_sample: int) -> dict:
    """The fp64 oracle, as it is, on a bounded sample of a large workload: the
    whole step on a canvas holding only the first n_sample masked positions
    of sequence 0 (the oracle's cost is linear in the masked positions it
    projects, so positions/s carries over to the whole batch)."""
    import numpy as np
    import oracle as O
    idx = np.nonzero(w.mask[0])[0][:n_sample]
    sub = np.zeros_like(w.mask)
    sub[0, idx] = 1
    t0 = time.perf_counter()
    O.score_commit(w.hidden, w.w_u, sub, w.cfg.dtype, P)
    t = time.perf_counter() - t0
    return {"value": len(idx) / t, "unit": "positions/s", "cores": blas_threads(), "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"one call of the step on the first {len(idx)} masked positions of sequence 0 only "
                      f"({len(idx)} of {w.n_masked} positions x {w.cfg.K} layers, V={w.cfg.V}, d={w.cfg.d}) in "
                      f"float64, {t:.1f} s; the oracle's cost is linear in the positions it projects"}


def time_calls(call, steps: int, warmup: int, event_every: int, flush=None):
    """Warm-up calls, then `steps` timed calls bracketed by events on the
    current stream (torch's, which the library launches on). Every
    `event_every`-th call also records events around the whole call and around
    the projection kernel (rpd_score_commit_timed). Returns (ms over all
    steps, projection ms per sampled call, call ms per sampled call); with a
    flush the steps' time is the sum of the sampled (every) calls."""
    import torch
    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    E = 1 if flush is not None else max(1, event_every)
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    nev = (steps + E - 1) // E
    proj_a, proj_b, call_a, call_b = ([ev() for _ in range(nev)] for _ in range(4))
    start, end = ev(), ev()
    for e in proj_a + proj_b + call_a + call_b:       # torch creates the HIP event at its first record
        e.record()
    torch.cuda.synchronize()
    assert all(e.cuda_event for e in proj_a + proj_b + call_a + call_b)
    start.record()
    for k in range(steps):
        if flush is not None:
            flush.fill_(k & 255)          # evicts W_U, hidden rows and outputs from the 256 MB cache
        if k % E == 0:
            j = k // E
            call(events=[call_a[j], proj_a[j], proj_b[j], None, call_b[j]])
        else:
            call()
    end.record()
    torch.cuda.synchronize()
    ms_total = start.elapsed_time(end)
    call_ms = [a.elapsed_time(b) for a, b in zip(call_a, call_b)]
    if flush is not None:    # the flushes are in the loop: time the calls alone
        ms_total = float(sum(call_ms))
    proj_ms = [a.elapsed_time(b) for a, b in zip(proj_a, proj_b)]
    return ms_total, proj_ms, call_ms


def roofline_entry(cfg, R: int, proj_ms_avg: float, step_ms: float, variant: str) -> dict:
    """Roofline of the projection kernel (algorithmic bytes or flops per launch
    over its event-timed average) and of the whole call (`call_frac`: the
    roofline time over the average time of a step in the timed loop)."""
    bytes_alg, flops_alg = proj_cost(cfg, R)
    t_bound = max(bytes_alg / (HBM_PEAK_GBS * 1e9), flops_alg / (MFMA_BF16_PEAK_TFLOPS * 1e12))
    if R < RIDGE_ROWS:
        achieved = bytes_alg / (proj_ms_avg / 1e3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4)}
    else:
        achieved = flops_alg / (proj_ms_avg / 1e3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4)}
    roof["traffic"] = read_traffic(variant, cfg.name)
    roof["kernel"] = f"{VARIANT_KERNEL[variant]} ({variant})"
    roof["kernel_us"] = round(proj_ms_avg * 1e3, 2)
    roof["call_frac"] = round(t_bound / (step_ms / 1e3), 4)
    roof["alg_bytes_per_launch"] = bytes_alg
    roof["alg_flops_per_launch"] = flops_alg
    return roof


def bench_mfma_regime(args, torch, rpd) -> dict:
    """The compute-bound regime beside the headline: the batched LLaDA-8B
    shape (8 sequences x 512 positions, 75% masked: 12,288 projected rows),
    timed like the headline (events around every call and its projection)."""
    import numpy as np
    from paper_2609_36452_amd.workload import CONFIGS, make_workload
    cfg = CONFIGS[args.mfma_config]
    log(f"mfma regime: drawing workload {cfg.name} seed {args.seed}")
    w = make_workload(cfg, args.seed)
    P = rpd.Params.strict(cfg.K, args.beta)
    dev = torch.device("cuda:0")
    hidden = torch.from_numpy(w.hidden).view(torch.bfloat16).to(dev)
    w_u = torch.from_numpy(w.w_u).view(torch.bfloat16).to(dev)
    mask = torch.from_numpy(w.mask).to(dev)
    call = rpd.ScoreCommit(hidden, w_u, mask, P, max_masked=w.n_masked)
    variant = rpd.projection_variant(cfg.K, cfg.B, cfg.L, cfg.d, cfg.V, hidden.dtype, max_masked=w.n_masked)
    K, W = args.mfma_steps, args.mfma_warmup
    log(f"  variant {variant}; warmup {W}, timing {K} calls")
    ms_total, proj_ms, call_ms = time_calls(call, K, W, 1)
    n, R = w.n_masked, w.n_masked * cfg.K
    ms_step = ms_total / K
    proj_avg = float(np.mean(proj_ms))
    log(f"  {ms_step * 1e3:.1f} us/step, projection {proj_avg * 1e3:.1f} us")
    pct = lambda xs: {f"p{q}": round(float(np.percentile(xs, q)) * 1e3, 2) for q in (10, 50, 90)}  # noqa: E731
    out = {
        "workload": f"{cfg.name}: d={cfg.d} V={cfg.V} B={cfg.B} L={cfg.L} K={cfg.K} masked={n} ({R} projected "
                    f"rows), rule=strict beta={P.beta}",
        "value": round(n * K / (ms_total / 1e3), 1),
        "unit": "positions/s",
        "steps": K,
        "warmup": W,
        "ms_per_step": round(ms_step, 5),
        "iterations_per_s": round(1e3 / ms_step, 2),
        "call_us_sampled": pct(call_ms),
        "projection_us_sampled": pct(proj_ms),
        "roofline": roofline_entry(cfg, R, proj_avg, ms_step, variant),
    }
    del call, hidden, mask
    if not args.no_cpu_baseline:
        import oracle as O
        log("  cpu baseline (oracle, sampled)")
        out["cpu_baseline"] = cpu_baseline_sampled(w, O.Params(**P.__dict__), args.mfma_cpu_positions)
    return out


def bench_library_gemm(args, torch, rpd) -> int:
    """Calibration, not the benchmark: the vendor library's plain bf16 GEMM
    (torch.mm, hipBLASLt) of the same masked rows against the same W_U, timed
    alternately with the projection of the commit step on the same data. The
    GEMM writes the R x V product and has no softmax; the projection writes
    per-tile softmax states only. One JSON line per workload."""
    import numpy as np
    from paper_2609_36452_amd.workload import CONFIGS, make_workload
    dev = torch.device("cuda:0")
    for name in args.library_gemm.split(","):
        cfg = CONFIGS[name]
        log(f"library gemm: drawing workload {cfg.name} seed {args.seed}")
        w = make_workload(cfg, args.seed)
        hidden = torch.from_numpy(w.hidden).view(torch.bfloat16).to(dev)
        w_u = torch.from_numpy(w.w_u).view(torch.bfloat16).to(dev)
        mask = torch.from_numpy(w.mask).to(dev)
        n, R = w.n_masked, w.n_masked * cfg.K
        pos = mask.reshape(-1).nonzero().reshape(-1)
        # the projected rows in the commit step's order: position-major, layer-minor
        x = hidden.reshape(cfg.K, -1, cfg.d)[:, pos].permute(1, 0, 2).reshape(R, cfg.d).contiguous()
        prod = torch.empty(R, cfg.V, dtype=torch.bfloat16, device=dev)
        call = rpd.ScoreCommit(hidden, w_u, mask, rpd.Params.strict(cfg.K, args.beta), max_masked=n)
        N = args.steps
        for _ in range(args.warmup):
            call()
            torch.mm(x, w_u.t(), out=prod)
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(N)]
        for e in ev:   # the binding records through HIP: each event needs its handle first
            for x_ in e:
                x_.record()
        torch.cuda.synchronize()
        for e in ev:
            call(events=[e[0], e[1], e[2], None, e[3]])
            e[4].record()
            torch.mm(x, w_u.t(), out=prod)
            e[5].record()
        torch.cuda.synchronize()
        t_proj = float(np.median([e[1].elapsed_time(e[2]) for e in ev])) * 1e3
        t_lib = float(np.median([e[4].elapsed_time(e[5]) for e in ev])) * 1e3
        fl = 2.0 * R * cfg.V * cfg.d
        print(json.dumps({
            "workload": cfg.name, "projected_rows": R, "d": cfg.d, "V": cfg.V, "calls": N,
            "projection_us_median": round(t_proj, 1), "library_gemm_us_median": round(t_lib, 1),
            "projection_tflops": round(fl / t_proj / 1e6, 1), "library_gemm_tflops": round(fl / t_lib / 1e6, 1),
            "projection_over_library": round(t_proj / t_lib, 4),
            "hbm_frac_projection": round((cfg.V * cfg.d * 2) / (t_proj * 1e-6) / (HBM_PEAK_GBS * 1e9), 4),
            "hbm_frac_library": round((cfg.V * cfg.d * 2) / (t_lib * 1e-6) / (HBM_PEAK_GBS * 1e9), 4)}), flush=True)
        del call, prod, x, hidden, w_u, mask
        torch.cuda.empty_cache()
    return 0


def proj_cost(cfg, rows: int):
    """Algorithmic HBM bytes and flops of one projection launch over ``rows``
    rows: W_U read once plus the rows, 2 flops per multiply-add."""
    el = 2 if cfg.dtype == "bf16" else 4
    return cfg.V * cfg.d * el + rows * cfg.d * el, 2.0 * rows * cfg.V * cfg.d


def decode_cpu_baseline(w, P, counts: list, budget_s: float) -> dict:
    """The oracle on the host: one whole call of the step on the fully masked
    first iteration, timed while it fits the budget, then scaled to a whole
    decode by the masked counts of the decode's iterations (the oracle's cost
    is proportional to the masked positions it projects)."""
    import oracle as O
    t, reps = 0.0, 0
    while reps == 0 or (t * (reps + 1) / reps < budget_s and reps < 64):
        t0 = time.perf_counter()
        pos, layer = O.layer_stats_masked(w.hidden, w.w_u, w.mask, w.cfg.dtype)
        O.assemble(w.mask, pos, layer, P)
        t += time.perf_counter() - t0
        reps += 1
    per_pos = t / reps / w.n_masked
    est = per_pos * sum(counts)
    return {"value": w.n_masked / est, "unit": "positions/s", "cores": blas_threads(), "kind": "oracle",
            "sample": f"{reps} whole call(s) of the step at the first iteration ({w.n_masked} masked positions x "
                      f"{w.cfg.K} layers, V={w.cfg.V}, d={w.cfg.d}) in float64, {t:.1f} s; scaled to the "
                      f"{sum(counts)} position-iterations of the decode"}


def bench_decode(args, w, P, hidden, w_u, mask, norm_kw) -> int:
    """Whole decodes: iterations of score-commit + canvas update until no
    position is masked, each decode from the same initial mask, HIP-graph
    replays with a read-back of the masked count every --sync-every
    iterations (the host has to learn when to stop)."""
    import numpy as np
    import torch
    from paper_2609_36452_amd import binding as rpd
    cfg = w.cfg
    # the decoder replays graphs unless a lazy call would read counts back (more than 256 masked)
    dec = rpd.Decoder(hidden, w_u, mask, P, graph=True, sync_every=args.sync_every, **norm_kw)
    log(f"decode warmup {args.warmup} (first decode captures the plans)")
    r = None
    for _ in range(max(args.warmup, 1)):
        dec.reset()
        r = dec.run()
    torch.cuda.synchronize()
    nfe, calls = r["iterations"], r["calls"]
    log(f"  NFE {nfe}, calls per decode {calls}, graphs captured {dec.captures}")
    K = args.steps
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    log(f"timing {K} decodes")
    t_wall0 = time.perf_counter()
    start.record()
    for _ in range(K):
        dec.reset()
        r = dec.run()
    end.record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall0
    ms_dec = start.elapsed_time(end) / K
    assert r["iterations"] == nfe
    # the same decode eagerly (launch by launch), for the launch overhead the graphs remove
    eager = rpd.Decoder(hidden, w_u, mask, P, graph=False, sync_every=args.sync_every, **norm_kw)
    eager.run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ke = max(1, min(K, 5))
    e0.record()
    for _ in range(ke):
        eager.reset()
        eager.run()
    e1.record()
    torch.cuda.synchronize()
    ms_eager = e0.elapsed_time(e1) / ke
    # projection time per iteration (stage events; eager)
    timed = rpd.Decoder(hidden, w_u, mask, P, graph=False, sync_every=args.sync_every, **norm_kw)
    rt = timed.run(stage_events=True)
    counts = [w.n_masked] + rt["left"][:-1]
    proj = rt["proj_ms"][:len(counts)]
    cls = {"hbm": [0.0, 0.0], "mfma": [0.0, 0.0]}
    sol = 0.0
    for n, ms in zip(counts, proj):
        by, fl = proj_cost(cfg, n * cfg.K)
        c = "hbm" if n * cfg.K < RIDGE_ROWS else "mfma"
        cls[c][0] += by if c == "hbm" else fl
        cls[c][1] += ms
        sol += max(by / (HBM_PEAK_GBS * 1e9), fl / (MFMA_BF16_PEAK_TFLOPS * 1e12)) * 1e3
    dom = max(cls, key=lambda c: cls[c][1])
    amount, ms_sum = cls[dom]
    if dom == "hbm":
        ach = amount / (ms_sum / 1e3) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4)}
    else:
        ach = amount / (ms_sum / 1e3) / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(ach / MFMA_BF16_PEAK_TFLOPS, 4)}
    roof["traffic"] = None
    roof["kernel"] = f"projection launches of the {dom}-bound iterations (varying variant)"
    # the lazy passes project only the rows still walking their suffix, a count the host never sees:
    # their rate is then stated against the eager work of the same iterations, not their own
    roof["work_basis"] = ("eager-equivalent: 2*K*n*V*d flops and V*d + K*n*d elements per iteration; the lazy "
                          "passes do less, so this overstates their own rate") if P.lazy else "algorithmic"
    roof["iterations"] = sum(1 for n in counts if (n * cfg.K < RIDGE_ROWS) == (dom == "hbm"))
    roof["kernel_ms_per_decode"] = round(ms_sum, 4)
    roof["projection_ms_per_decode"] = round(float(np.sum(proj)), 4)
    roof["speed_of_light_frac"] = round(sol / float(np.sum(proj)), 4)
    value = w.n_masked / (ms_dec / 1e3)
    log(f"  {ms_dec:.3f} ms/decode (eager {ms_eager:.3f}), {nfe / ms_dec * 1e3:.0f} iterations/s, wall {t_wall:.2f} s")
    out = {
        "metric": "positions decoded/sec over whole decodes at LLaDA-8B shape (score-commit + canvas update "
                  "per iteration until no mask)",
        "value": round(value, 1),
        "unit": "positions/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_dec, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded random W_U ~ N(0,1/d) and hidden states of the model shape, held fixed "
                "between iterations)",
        "config": {"workload": f"{cfg.name} decode: d={cfg.d} V={cfg.V} B={cfg.B} L={cfg.L} K={cfg.K} "
                               f"{w.n_masked} masked at the start, rule={args.rule} beta={P.beta}"
                               + (f" block={P.block}" if P.block else ""),
                   "nfe": nfe, "calls_per_decode": calls, "sync_every": args.sync_every,
                   "graphs": dec.captures, "commit_rule": "rpd_block" if P.block else "rpd",
                   "final_norm": bool(args.norm), "lazy_projection": bool(P.lazy)},
        "iterations_per_s": round(nfe / ms_dec * 1e3, 1),
        "eager_ms_per_step": round(ms_eager, 5),
        "roofline": roof,
    }
    if not args.no_cpu_baseline and not args.norm:
        import oracle as O
        log("cpu baseline (oracle)")
        out["cpu_baseline"] = decode_cpu_baseline(w, O.Params(**P.__dict__), counts, args.cpu_budget)
    print(json.dumps(out), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default=None,
                    help="workload (default llada_late; llada_100, a fully masked canvas, with --decode)")
    ap.add_argument("--seed", type=int, default=1)
    ap.add_argument("--rule", default="strict", choices=["strict", "llada", "dream", "llada_block"],
                    help="commit rule: strict agreement (default), the paper's LLaDA / Dream settings, or "
                         "RPD-block with the LLaDA settings and blocks of 32")
    ap.add_argument("--beta", type=float, default=1.0)
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--lazy", action="store_true",
                    help="lazy layerwise projection (intermediate layers only where stability decides)")
    ap.add_argument("--norm", action="store_true",
                    help="pass a normalization gain: layers 0..K-2 go through the final normalization first")
    ap.add_argument("--no-copy-probe", action="store_true",
                    help="skip the plain copy kernel of known size that runs after the timed region (it scales "
                         "the HBM byte counters and gives this GPU's copy bandwidth as context)")
    ap.add_argument("--copy-probe", action="store_true", help=argparse.SUPPRESS)   # the default; kept for old commands
    ap.add_argument("--decode", action="store_true",
                    help="time whole decodes instead of single calls: score-commit and canvas update per "
                         "iteration until no position is masked (HIP-graph replays)")
    ap.add_argument("--sync-every", type=int, default=8,
                    help="--decode: iterations between read-backs of the masked count")
    ap.add_argument("--cold", action="store_true",
                    help="flush the last-level cache between calls with a 512 MB write (not timed: every call "
                         "carries events and the value comes from the per-call times)")
    ap.add_argument("--mfma-config", default="llada_batched",
                    help="the compute-bound workload timed beside the headline in the same line (mfma_regime); "
                         "empty to skip")
    ap.add_argument("--mfma-steps", type=int, default=20)
    ap.add_argument("--mfma-warmup", type=int, default=5)
    ap.add_argument("--mfma-cpu-positions", type=int, default=384,
                    help="masked positions of the oracle's sample for the mfma_regime CPU baseline")
    ap.add_argument("--library-gemm", default=None, metavar="CONFIGS",
                    help="calibration only: time the vendor library's bf16 GEMM (torch.mm) of the same rows "
                         "beside the projection, for each comma-separated workload, and print one JSON line each")
    ap.add_argument("--event-every", type=int, default=10,
                    help="record the projection's HIP events on every N-th timed call (each event record "
                         "costs the stream a few microseconds; a sampled call measured about 9 us slower)")
    args = ap.parse_args()
    if args.config is None:
        args.config = "llada_100" if args.decode else "llada_late"
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the commit step is benchmarked on a single MI355X "
              f"(--gpus {args.gpus} is not supported)", file=sys.stderr)
        return 2

    import numpy as np
    import torch
    from paper_2609_36452_amd import binding as rpd
    from paper_2609_36452_amd.workload import CONFIGS, make_workload

    if not os.path.exists(rpd._LIB_PATH):
        from paper_2609_36452_amd.build import build
        build()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.library_gemm:
        return bench_library_gemm(args, torch, rpd)
    cfg = CONFIGS[args.config]
    log(f"drawing workload {cfg.name} seed {args.seed}")
    t0 = time.perf_counter()
    w = make_workload(cfg, args.seed)
    log(f"  drawn in {time.perf_counter() - t0:.1f} s; masked positions {w.n_masked}")
    if args.rule == "strict":
        P = rpd.Params.strict(cfg.K, args.beta)
    elif args.rule == "llada":
        P = rpd.Params.llada()
    elif args.rule == "llada_block":
        P = dataclasses.replace(rpd.Params.llada(), block=32)
    else:
        P = rpd.Params.dream()
    if args.lazy:
        P = dataclasses.replace(P, lazy=True)
    dev = torch.device("cuda:0")
    if cfg.dtype == "bf16":
        hidden = torch.from_numpy(w.hidden).view(torch.bfloat16).to(dev)
        w_u = torch.from_numpy(w.w_u).view(torch.bfloat16).to(dev)
    else:
        hidden = torch.from_numpy(w.hidden).to(dev)
        w_u = torch.from_numpy(w.w_u).to(dev)
    mask = torch.from_numpy(w.mask).to(dev)
    norm_kw = {}
    if args.norm:
        from paper_2609_36452_amd.workload import round_bf16_bits
        g = np.random.default_rng(args.seed + 7).uniform(0.5, 2.0, cfg.d)
        gt = torch.from_numpy(round_bf16_bits(g)).view(torch.bfloat16) if cfg.dtype == "bf16" else \
            torch.from_numpy(g.astype(np.float32))
        norm_kw = dict(norm_weight=gt.to(dev), norm_eps=1e-5)
    if args.decode:
        return bench_decode(args, w, P, hidden, w_u, mask, norm_kw)
    call = rpd.ScoreCommit(hidden, w_u, mask, P, max_masked=w.n_masked, **norm_kw)
    variant = rpd.projection_variant(cfg.K, cfg.B, cfg.L, cfg.d, cfg.V, hidden.dtype, max_masked=w.n_masked)
    log(f"projection variant {variant}")
    torch.cuda.synchronize()
    K = args.steps
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev) if args.cold else None
    log(f"warmup {args.warmup}, timing {K} steps")
    t_wall0 = time.perf_counter()
    ms_total, proj_ms, call_ms = time_calls(call, K, args.warmup, args.event_every, flush)
    t_wall = time.perf_counter() - t_wall0
    ms_step = ms_total / K
    proj_avg = float(np.mean(proj_ms))
    pct = lambda xs: {f"p{q}": round(float(np.percentile(xs, q)) * 1e3, 2) for q in (10, 50, 90)}  # noqa: E731
    n = w.n_masked
    R = n * cfg.K
    value = n * K / (ms_total / 1e3)
    log(f"  {ms_step * 1e3:.1f} us/step, projection {proj_avg * 1e3:.1f} us (median "
        f"{np.median(proj_ms) * 1e3:.1f}), wall {t_wall:.3f} s")
    roof = roofline_entry(cfg, R, proj_avg, ms_step, variant)
    roof["timed_launches"] = len(proj_ms)

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "positions/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded random W_U ~ N(0,1/d) and hidden states of the model shape)",
        "config": {"workload": f"{cfg.name}: d={cfg.d} V={cfg.V} B={cfg.B} L={cfg.L} K={cfg.K} "
                               f"masked={n} ({R} projected rows), rule={args.rule} beta={P.beta}"
                               + (f" block={P.block}" if P.block else ""),
                   "masked_positions": n, "projected_rows": R, "seed": args.seed,
                   "commit_rule": "rpd_block" if P.block else "rpd", "final_norm": bool(args.norm),
                   "lazy_projection": bool(P.lazy),
                   "cache_state": ("cold: a 512 MB write between calls evicts everything; value from per-call "
                                   "events" if args.cold else
                                   "W_U streamed from HBM every call (larger than the 256 MB last-level cache); "
                                   "hidden rows, mask and outputs warm from the previous call")},
        "iterations_per_s": round(1e3 / ms_step, 1),
        "call_us_sampled": pct(call_ms),
        "projection_us_sampled": pct(proj_ms),
        "roofline": roof,
    }
    del call
    if not args.no_copy_probe:
        out["copy_probe_gbs"] = round(copy_probe(torch), 1)
    if not args.no_cpu_baseline and not args.norm:
        import oracle as O
        OP = O.Params(**P.__dict__)
        log("cpu baseline (oracle)")
        out["cpu_baseline"] = cpu_baseline(w, OP, args.cpu_budget)
    if args.mfma_config and args.mfma_config != cfg.name and not args.norm and not args.lazy and not args.cold:
        out["mfma_regime"] = bench_mfma_regime(args, torch, rpd)
    out["paper_context"] = PAPER_CONTEXT
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
