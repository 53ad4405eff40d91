#!/usr/bin/env python3
"""Benchmark of the LAM hot path on one MI355X.

One step is one pass of the whole hot path over synthetic inputs shaped like
the paper's workloads:
  1. Q_eps encode + decode of 2^26 float32 values (half N(0, 0.04^2), half
     U(-1, 1)) at eps = 1e-3 with a declared absmax of 1 (10-bit codes); four
     input sets rotate so that no pass reads from the 256 MB last-level cache;
  2. the greedy near-duplicate test over the 27,986-row subset stream (600
     trajectories of ~47 chunks, D = 768) in batches of 1,024, tau = 0.95,
     into a cleared store (calls that do not wait for the device);
  3. Q_eps of the retained store at eps = 1e-3 (absmax measured on the GPU),
     and its decode;
  4. top-10 scoring of 1,024 queries against the quantized store.
value = near-duplicate pairs per second of the whole step, counting the
algorithmic pairs of exhaustive greedy (each arrival against every row
retained at its arrival: config.pairs_per_step).  The screen's roofline counts
the pairs its launches screen (each chunk against the rows retained before the
chunk, plus the chunk's own lower triangle: config.screened_pairs_per_step).

Usage: python bench.py [--steps K] [--warmup W] [--no-cpu-baseline] [--no-extras] [--band-grid]
Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
MFMA_F16_PEAK_TFLOPS = 2500.0  # MI355X dense fp16 matrix, published
D = 768
EPS = 1e-3
TAU = 0.95
BATCH = 1024
TOPK = 10
RAW_LOG2N = 26
RAW_SETS = 4
BAND_R = 4          # band width and quantizer step (eps = rel * sigma, sigma = 1 / sqrt(D))
BAND_REL = 0.2      # of the banded candidate index, the operating point for tau = 0.95
BAND_REPS = 5
BAND_PREFIX = 4096  # arrivals of the grid's trial run per setting
QEPS_WIDTH_EPS = (1e-2, 1e-3, 1e-4)   # 7-, 10- and 14-bit codes of the raw workload
TRIAD_N = 1 << 27                     # floats per triad array (3 x 512 MB)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip timing the CPU oracle")
    ap.add_argument("--band-grid", action="store_true",
                    help="instead of the step: the banded candidate index over band widths 2..32 and steps "
                         "0.01..0.3 sigma on the subset stream (one JSON line)")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the measurements beside the step (removal ceiling, certificate, block codec, "
                         "banded stream), so that a profiler sees the steps only")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed steps, run a plain 1 GiB device-to-device copy three times (a "
                         "known-size reference for hardware byte counters)")
    return ap.parse_args()


KERNELS = ("qeps_encode", "qeps_decode", "dedup_prep", "dedup_screen", "dedup_verify", "dedup_resolve_append",
           "dedup_resolve", "dedup_append", "store_encode", "store_decode", "score_prep", "score_sample",
           "score_mfma", "score_merge", "score_fallback")
HERE = os.path.dirname(os.path.abspath(__file__))
TRAFFIC_FILE = os.path.join(HERE, "profiles", "traffic.json")


def _sha256(path):
    import hashlib
    with open(os.path.join(HERE, path), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    runs (FETCH_SIZE and WRITE_SIZE, each scaled by what the counter reads for a
    plain copy of known size), or None when there are none or the kernel's
    sources have changed since they were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
        k = t["kernels"][kernel]
        if any(_sha256(p) != h for p, h in k["sources"].items()):
            return None
        cal = t["copy_calibration"]
        ff = cal["bytes"] / 1024.0 / cal["fetch_kib"]
        wf = cal["bytes"] / 1024.0 / cal["write_kib"]
        return (k["fetch_kib_per_dispatch"] * ff + k["write_kib_per_dispatch"] * wf) * 1024.0
    except (OSError, KeyError, ValueError):
        return None


def cpu_baseline(x, pairs, raw, q):
    """The oracle, as it stands, on the host's cores: the whole subset stream
    through the dedup oracle (the headline figure), and beside it Q_eps encode
    on a 2^24-value prefix of the raw workload and top-10 scoring of 256
    queries against the stream's retained rows coded by the oracle."""
    import numpy as np
    from oracle import dedup, qeps, score
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    t0 = time.perf_counter()
    r = dedup.greedy(x, TAU, block=512)
    dt = time.perf_counter() - t0
    out = {"value": pairs / dt / 1e6, "unit": "M pairs/s", "cores": int(threads), "kind": "oracle",
           "seconds": dt,
           "sample": f"exhaustive greedy over the whole {x.shape[0]}-row subset stream (ingest only; "
                     f"binary64 BLAS screen + exact rational ties)"}
    xs = raw[:1 << 24]
    t0 = time.perf_counter()
    _, _, plan = qeps.encode(xs, EPS, absmax=1.0)
    dq = time.perf_counter() - t0
    nbytes = (4 + plan["bits"] / 8) * xs.size
    out["qeps_encode"] = {"value": nbytes / dq / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle", "seconds": dq,
                          "sample": f"2^24 values of the raw workload at eps={EPS} ({plan['bits']}-bit codes; "
                                    f"binary64 NumPy + exact rational near-ties, one thread)"}
    store_ids = r["kept"]
    store_codes = qeps.codes(x[store_ids], EPS).reshape(store_ids.size, -1)   # not timed
    qs = q[:256]
    t0 = time.perf_counter()
    score.score_topk(qs, store_codes, store_ids, EPS, TOPK)
    dsc = time.perf_counter() - t0
    out["scoring"] = {"value": qs.shape[0] / dsc, "unit": "queries/s", "cores": int(threads), "kind": "oracle",
                      "seconds": dsc,
                      "sample": f"{qs.shape[0]} queries top-{TOPK} against the {store_codes.shape[0]}-row quantized "
                                f"store of the stream (binary64 BLAS scores + sort)"}
    return r, out


def banded_ingest(lam, torch, np, xd, rep_exh, pairs, ctx, r=BAND_R, rel=BAND_REL, reps=BAND_REPS,
                  screened=True):
    """The subset stream through a store with the banded candidate index
    (band width r, step eps = rel / sqrt(D)) next to the screened store:
    candidate pairs against the exhaustive pair count, removal and agreement
    with exhaustive greedy, and the time of a whole-stream ingest (calls that
    do not wait) for both stores."""
    n = xd.shape[0]
    eps = rel / D ** 0.5
    band = lam.Store(D, TAU, n, ctx=ctx, eps_band=eps, band_width=r)
    outs = [torch.empty(min(BATCH, n - b0), dtype=torch.int64, device=xd.device) for b0 in range(0, n, BATCH)]

    def stream(s, sync):
        s.clear()
        st = [s.ingest(xd[b0:b0 + BATCH], rep=outs[bi], sync=sync)[1] for bi, b0 in enumerate(range(0, n, BATCH))]
        s.info()   # waits for calls that did not wait
        return st

    stats = stream(band, True)
    brep = torch.cat(outs).cpu().numpy()
    cand = sum(st["n_ambiguous_pairs"] for st in stats)
    stores = [("banded", band)] + ([("screened", lam.Store(D, TAU, n, ctx=ctx))] if screened else [])
    times = {}
    for name, s in stores:
        stream(s, False)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            stream(s, False)
        torch.cuda.synchronize()
        times[name] = (time.perf_counter() - t0) * 1e3 / reps
    kept = int(np.count_nonzero(brep < 0))
    dropped_exh = int(np.count_nonzero(rep_exh >= 0))
    out = {"band_width": r, "eps_band": eps, "rel": rel,
           "candidate_pairs": int(cand), "exhaustive_pairs": int(pairs), "candidate_frac": cand / pairs,
           "kept": kept, "removal": 1.0 - kept / n, "removal_recall": (n - kept) / max(dropped_exh, 1),
           "rep_agreement": float(np.mean(brep == rep_exh)),
           "rep_equal_to_exhaustive": bool(np.array_equal(brep, rep_exh)), "ms_per_stream": times["banded"]}
    if screened:
        out["screened_ms_per_stream"] = times["screened"]
    del band
    return out


def beside_the_step(lam, torch, np, xd, qd, store, rep, pairs, ctx, raw_sets, raw_out, width_codes):
    """Measurements beside the timed step (not in it): the decision
    statistics of the stream (ambiguous pairs, exact decisions, smallest
    decided margin), the triad and matrix-unit anchors, raw Q_eps at three widths,
    the stream as one ingest call, the screen at scale, the large online store at full size, the tiny
    workload's per-call latency, the removal ceiling of the stream, the share
    of benchmark queries whose top-10 is certified rank-invariant, the
    per-block codec (size and speed) on the retained store, scoring at the
    corpus size, and the stream through the banded candidate index."""
    # first, before the heavy measurements below: run after them, the 7-bit
    # decode took 94 us per launch against 65 us in a process of its own
    widths = qeps_widths(lam, torch, raw_sets, raw_out, width_codes, ctx, None)
    ceil = lam.removal_ceiling(xd, TAU, batch=BATCH, ctx=ctx)
    cert = store.score_topk_certified(qd, TOPK)[3]
    blk_t = block_codec_timing(lam, torch, store, ctx)
    blk = store.block_encode()
    triad = triad_anchor(lam, torch, ctx)
    for row in widths.values():
        for name in ("qeps_encode", "qeps_decode"):
            row[name]["frac_of_triad"] = row[name]["GBps"] / triad["GBps"]
    matmul = matmul_anchor(torch)
    # the stream once more with calls that wait, for the decision statistics
    n = xd.shape[0]
    probe = lam.Store(D, TAU, n, ctx=ctx)
    st = [probe.ingest(xd[b0:b0 + BATCH])[1] for b0 in range(0, n, BATCH)]
    decisions = {"ambiguous_pairs": int(sum(t["n_ambiguous_pairs"] for t in st)),
                 "exact_escalations": int(sum(t["n_exact_escalations"] for t in st)),
                 "min_margin_d2": float(min(t["min_margin_d2"] for t in st))}
    del probe
    steady = screen_steady_state(lam, torch, np, ctx)
    small = screen_steady_state(lam, torch, np, ctx, policy="small")
    steady["small_tile"] = {k: small[k] for k in ("tile", "screen_ms_per_call", "screen_TFLOPs", "screen_frac_of_peak")}
    steady["screen_frac_of_matmul_anchor"] = steady["screen_TFLOPs"] / matmul["TFLOPs"]
    steady["screen_frac_of_matmul_anchor_k768"] = steady["screen_TFLOPs"] / matmul["TFLOPs_k768_nt"]
    return {"decisions": decisions,
            "triad": triad,
            "matmul_anchor": matmul,
            "qeps_widths": widths,
            "screen_steady_state": steady,
            "one_call": one_call_ingest(lam, torch, np, xd, rep, pairs, ctx),
            "online_store": online_store_run(lam, torch, np, ctx),
            "tiny_latency": tiny_latency(lam, torch, ctx),
            "corpus_scoring": corpus_scoring(lam, torch, np, ctx),
            "removal_ceiling": {k: ceil[k] for k in ("kept", "kept_2delta", "removal", "ceiling",
                                                     "frac_of_ceiling", "bits_lo", "bits_hi")},
            "certified_top10_frac": float(cert.float().mean().item()),
            "block_codec": {**{k: blk[k] for k in ("bits_per_code", "plain_bits", "codec_ratio", "composite_ratio")},
                            **{k: v for k, v in blk_t.items() if k.startswith("store_block")}},
            "banded": banded_ingest(lam, torch, np, xd, rep, pairs, ctx)}


def one_call_ingest(lam, torch, np, xd, rep_step, pairs, ctx, reps=5):
    """The subset stream as a single ingest call: the library walks it in
    chunks of 4,096 rows, each screened against the rows retained before it
    and resolved in arrival order, so the decisions equal those of the step's
    28 calls of 1,024.  Wall time of the call (inputs resident, store created
    beforehand), best of `reps`."""
    n = xd.shape[0]
    out = torch.empty(n, dtype=torch.int64, device=xd.device)
    times = []
    for _ in range(reps):
        s = lam.Store(D, TAU, n, ctx=ctx)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        s.ingest(xd, rep=out, sync=False)
        torch.cuda.synchronize()
        times.append(time.perf_counter() - t0)
        del s
    ms = min(times) * 1e3
    return {"workload": f"subset stream as one call of {n} rows (chunks of 4,096 inside the call)", "ms": ms,
            "M_pairs_per_s": pairs / (ms / 1e3) / 1e6,
            "rep_equal_to_step": bool(np.array_equal(out.cpu().numpy(), rep_step))}


def corpus_scoring(lam, torch, np, ctx, calls=5):
    """Scoring at the corpus size: 4,096 queries top-10 against all 361,802
    records of the corpus recipe at D = 768 (every record in the store,
    quantized at eps = 1e-3).  Work is 2 D flop per (query, row)."""
    import synth
    cfg = synth.corpus_retrieval()
    xd = torch.from_numpy(cfg["x"]).cuda()
    qd = torch.from_numpy(cfg["q"]).cuda()
    n, nq = xd.shape[0], qd.shape[0]
    s = lam.Store(D, 1.0, n, ctx=ctx)
    for b0 in range(0, n, 16384):
        s.ingest(xd[b0:b0 + 16384], sync=False)
    p = s.quantize(cfg["eps"])
    out = s.score_topk(qd, cfg["k"])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(calls):
        s.score_topk(qd, cfg["k"], out=out)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / calls
    flops = 2.0 * D * nq * s.size
    del s, xd
    return {"workload": f"corpus recipe: {nq} queries top-{cfg['k']} against {n} rows, D = {D}, "
                        f"{p.bits}-bit codes", "ms_per_call": ms, "queries_per_s": nq / (ms / 1e3),
            "TFLOPs_algorithmic": flops / (ms / 1e3) / 1e12,
            "frac_of_peak": flops / (ms / 1e3) / 1e12 / MFMA_F16_PEAK_TFLOPS}


def screen_steady_state(lam, torch, np, ctx, m=262_144, batch=4096, calls=5, policy="auto"):
    """The screen at scale (D = 768): calls of 4,096 arrivals against the
    store left by ingesting 262,144 rows of the online-store recipe at D = 768
    (clusters of ~51, 20 % planted copies; drawn on the device).  Pairs are
    the algorithmic pairs of the measured calls.  policy: the screen's tile
    (lam_ctx_set_screen_tile; "auto" takes the 256 x 256 tile at this size)."""
    import synth
    cfg = synth.online_store_device(seed=6, n=m + calls * batch, n_clusters=m // 51, d=D, nq=16)
    x = cfg["x"]
    ctx.set_screen_tile(policy)
    s = lam.Store(D, TAU, x.shape[0], ctx=ctx)
    for b0 in range(0, m, batch):
        s.ingest(x[b0:b0 + batch], sync=False)
    sizes, pairs = [], 0
    size0 = s.info().size
    torch.cuda.synchronize()
    ctx.profile_reset()
    ctx.profile_only("dedup_screen")
    ctx.profile(True)
    t0 = time.perf_counter()
    for c in range(calls):
        b0 = m + c * batch
        _, st = s.ingest(x[b0:b0 + batch])       # waits: one call at a time
        sizes.append(st["store_size"])
    t1 = time.perf_counter()
    ctx.profile(False)
    ctx.profile_only(None)
    ctx.set_screen_tile("auto")
    tot_ms, cnt = ctx.profile_read("dedup_screen")
    before = [size0] + sizes[:-1]
    pairs = sum(batch * k + batch * (batch - 1) // 2 for k in before)
    flops = 2.0 * D * pairs
    # the automatic choice: 256 x 256 from 768 such tiles in the launch
    large = policy == "large" or (policy == "auto" and
                                  ((size0 + 255) // 256) * (batch // 256) + (batch // 256) * (batch // 256 + 1) // 2 >= 768)
    return {"workload": f"online-store recipe at D = {D}: {batch}-row batches against {size0} retained rows",
            "tile": "256x256" if large else "128x128",
            "calls": calls, "pairs": pairs, "ms_per_call": (t1 - t0) * 1e3 / calls,
            "screen_ms_per_call": tot_ms / max(cnt, 1),
            "M_pairs_per_s": pairs / (t1 - t0) / 1e6,
            "screen_TFLOPs": flops / (tot_ms / 1e3) / 1e12,
            "screen_frac_of_peak": flops / (tot_ms / 1e3) / 1e12 / MFMA_F16_PEAK_TFLOPS}


def triad_anchor(lam, torch, ctx, reps=20):
    """The bandwidth anchor: triad c = a + s b over 3 x 512 MB float32
    (lam_triad), timed by its launches; 12 bytes per element."""
    a = torch.ones(TRIAD_N, dtype=torch.float32, device="cuda")
    b = torch.full((TRIAD_N,), 2.0, dtype=torch.float32, device="cuda")
    c = torch.empty_like(a)
    lam.triad(a, b, c, 3.0, ctx=ctx)
    torch.cuda.synchronize()
    ctx.profile_reset()
    ctx.profile_only("triad")
    ctx.profile(True)
    for _ in range(reps):
        lam.triad(a, b, c, 3.0, ctx=ctx)
    torch.cuda.synchronize()
    ctx.profile(False)
    ctx.profile_only(None)
    tot, cnt = ctx.profile_read("triad")
    ok = bool(torch.all(c == 7.0).item())
    del a, b, c
    gbs = 12.0 * TRIAD_N / (tot / cnt / 1e3) / 1e9
    return {"workload": "triad c = a + 3 b, 3 x 512 MB float32", "GBps": gbs, "frac_of_spec": gbs / HBM_PEAK_GBS,
            "us_per_launch": tot / cnt * 1e3, "result_checked": ok}


def matmul_anchor(torch, n=8192, reps=10):
    """The matrix-unit anchor: an n^3 fp16 GEMM with float32 accumulation
    through the vendor BLAS (torch.matmul) on N(0, 1) operands, the fp16
    matmul row of the paper's anchors (App. "Measured hardware constants",
    Table "anchors": an 8192^3 GEMM).  A measurement, not a step of the path."""
    def timed(a, b):
        for _ in range(3):
            c = torch.matmul(a, b)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            c = torch.matmul(a, b)
        e1.record()
        e1.synchronize()
        del c
        return e0.elapsed_time(e1) / reps

    g = torch.Generator(device="cuda").manual_seed(5)
    a = torch.randn(n, n, device="cuda", dtype=torch.float16, generator=g)
    b = torch.randn(n, n, device="cuda", dtype=torch.float16, generator=g)
    ms = timed(a, b)
    # at the screen's reduction depth, K = 768, both operands K-major (C = A B^T)
    ak = torch.randn(32768, 768, device="cuda", dtype=torch.float16, generator=g)
    bk = torch.randn(32768, 768, device="cuda", dtype=torch.float16, generator=g)
    ms768 = timed(ak, bk.t())
    del ak, bk
    torch.cuda.empty_cache()
    # the same GEMM on all-zero operands: the matrix units' rate depends on
    # the operand data (switching activity), so the anchor uses random data
    a.zero_()
    b.zero_()
    ms0 = timed(a, b)
    del a, b
    tf = 2.0 * n ** 3 / (ms / 1e3) / 1e12
    return {"workload": f"fp16 GEMM {n}^3 (torch.matmul), N(0, 1) operands", "ms": ms, "TFLOPs": tf,
            "frac_of_spec": tf / MFMA_F16_PEAK_TFLOPS, "TFLOPs_zero_operands": 2.0 * n ** 3 / (ms0 / 1e3) / 1e12,
            "TFLOPs_k768_nt": 2.0 * 32768 * 32768 * 768 / (ms768 / 1e3) / 1e12,
            "k768_workload": "fp16 GEMM 32768 x 32768 x 768, C = A B^T (both K-major), N(0, 1) operands"}


def qeps_widths(lam, torch, raw_sets, raw_out, width_codes, ctx, triad_gbs, reps=20):
    """Raw Q_eps (2^26 values) at eps = 1e-2, 1e-3 and 1e-4 (7-, 10- and
    14-bit codes, absmax 1 declared): encode and decode GB/s from events the
    launches stamp themselves, four input sets rotating; (4 + b/8) bytes per
    element, against the spec and the measured triad.  The code buffers
    (width_codes, sized for the widest codes) are allocated with the other
    inputs at the start: buffers allocated after the other measurements had
    freed memory landed where the 7-bit decode ran at half its rate."""
    n = raw_sets[0].numel()
    out = {}
    for eps in QEPS_WIDTH_EPS:
        p = lam.qeps_plan(eps, 1.0, "bits", n)
        codes = [w[:p.code_bytes // 4] for w in width_codes]
        for k in range(len(raw_sets)):   # warm-up
            lam.quantize(raw_sets[k], eps, absmax=1.0, out=codes[k], ctx=ctx)
            lam.dequantize(codes[k], p, out=raw_out[k], ctx=ctx)
        torch.cuda.synchronize()
        ctx.profile_reset()
        ctx.profile_only("qeps_encode,qeps_decode")
        ctx.profile(True)
        for i in range(reps):
            k = i % len(raw_sets)
            lam.quantize(raw_sets[k], eps, absmax=1.0, out=codes[k], ctx=ctx)
            lam.dequantize(codes[k], p, out=raw_out[k], ctx=ctx)
        torch.cuda.synchronize()
        ctx.profile(False)
        ctx.profile_only(None)
        nbytes = (4 + p.bits / 8) * n
        row = {"bits": int(p.bits)}
        for name in ("qeps_encode", "qeps_decode"):
            tot, cnt = ctx.profile_read(name)
            gbs = nbytes / (tot / cnt / 1e3) / 1e9
            row[name] = {"us_per_launch": tot / cnt * 1e3, "GBps": gbs, "frac_of_spec": gbs / HBM_PEAK_GBS,
                         "frac_of_triad": gbs / triad_gbs if triad_gbs else None}
        out[f"eps={eps:g}"] = row
        del codes
    return out


def online_store_run(lam, torch, np, ctx, calls=2):
    """The large online store at its full size: 1,048,576 rows of D = 1,024
    (16,384 clusters, 20 % planted copies; drawn on the device) ingested in
    batches of 4,096 with calls that do not wait, tau = 0.95; the store coded
    at eps = 1e-3; then 16,384 queries top-50.  The screen is timed by its own
    launches; pairs are the algorithmic (retained at arrival) and the screened
    ones."""
    import synth
    cfg = synth.online_store_device(device="cuda")
    x, q = cfg["x"], cfg["q"]
    n, d = x.shape
    batch, k, eps = cfg["batch"], cfg["k"], cfg["eps"]
    s = lam.Store(d, cfg["tau"], n, ctx=ctx)
    reps = [torch.empty(min(batch, n - b0), dtype=torch.int64, device="cuda") for b0 in range(0, n, batch)]
    ingest_s = []
    for c in range(calls):
        s.clear()
        torch.cuda.synchronize()
        if c == calls - 1:
            ctx.profile_reset()
            ctx.profile_only("dedup_screen")
            ctx.profile(True)
        t0 = time.perf_counter()
        for bi, b0 in enumerate(range(0, n, batch)):
            s.ingest(x[b0:b0 + batch], rep=reps[bi], sync=False)
        info = s.info()   # waits for every call
        ingest_s.append(time.perf_counter() - t0)
    ctx.profile(False)
    ctx.profile_only(None)
    scr_ms, scr_n = ctx.profile_read("dedup_screen")
    rep = torch.cat(reps)
    kept = (rep < 0).to(torch.int64)
    kept_before = torch.cumsum(kept, 0) - kept
    pairs = int(kept_before.sum().item())
    starts = torch.arange(0, n, batch, device="cuda")
    nb = torch.clamp(n - starts, max=batch)
    screened = int((nb * kept_before[starts]).sum().item() + (nb * (nb - 1) // 2).sum().item())
    t0 = time.perf_counter()
    p = s.quantize(eps)
    q_ms = (time.perf_counter() - t0) * 1e3
    res = s.score_topk(q, k)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(3):
        s.score_topk(q, k, out=res)
    torch.cuda.synchronize()
    sc_ms = (time.perf_counter() - t0) * 1e3 / 3
    t_ing = min(ingest_s)
    flops = 2.0 * d * screened
    out = {"workload": f"online store: {n} x {d} in batches of {batch}, tau={cfg['tau']}, eps={eps}, "
                       f"{q.shape[0]} queries top-{k}",
           "kept": int(info.size), "ingest_s": t_ing, "M_pairs_per_s": pairs / t_ing / 1e6, "pairs": pairs,
           "screened_pairs": screened, "screen_ms": scr_ms, "screen_launches": scr_n,
           "screen_TFLOPs": flops / (scr_ms / 1e3) / 1e12,
           "screen_frac_of_peak": flops / (scr_ms / 1e3) / 1e12 / MFMA_F16_PEAK_TFLOPS,
           "store_quantize_ms": q_ms, "store_code_bits": int(p.bits),
           "scoring_ms": sc_ms, "queries_per_s": q.shape[0] / (sc_ms / 1e3),
           "scoring_TFLOPs_algorithmic": 2.0 * d * q.shape[0] * info.size / (sc_ms / 1e3) / 1e12}
    del s, x, q, reps, rep
    return out


def tiny_latency(lam, torch, ctx, calls=20):
    """The tiny workload as a latency test: 4,096 rows of D = 768 ingested as
    four calls of 1,024 that each wait (median ms per call, host to host),
    the store coded, and 64 queries top-10 (median ms per scoring call that
    waits)."""
    import synth
    t = synth.tiny_ingest()
    x = torch.from_numpy(t["x"]).cuda()
    q = torch.from_numpy(t["q"]).cuda()
    s = lam.Store(x.shape[1], t["tau"], x.shape[0], ctx=ctx)
    per_call = []
    for c in range(calls // 4 + 1):
        s.clear()
        torch.cuda.synchronize()
        for b0 in range(0, x.shape[0], 1024):
            t0 = time.perf_counter()
            s.ingest(x[b0:b0 + 1024])   # waits
            per_call.append((time.perf_counter() - t0) * 1e3)
    s.quantize(t["eps"])
    out = s.score_topk(q, 10)
    sc = []
    for _ in range(calls):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        s.score_topk(q, 10, out=out)
        torch.cuda.synchronize()
        sc.append((time.perf_counter() - t0) * 1e3)
    per_call = sorted(per_call[4:])   # the first pass warms up
    sc.sort()
    return {"workload": "tiny ingest: 4096 x 768 in calls of 1024 that wait; 64 queries top-10",
            "ingest_ms_per_call_p50": per_call[len(per_call) // 2], "ingest_ms_per_call_p90": per_call[int(0.9 * len(per_call))],
            "scoring_ms_p50": sc[len(sc) // 2], "scoring_ms_p90": sc[int(0.9 * len(sc))], "kept": int(s.size)}


def block_codec_timing(lam, torch, store, ctx, reps=10):
    """The per-block codec on the benchmark's store: encode (widths, then bit
    planes), decode to float32 and expansion back to the fixed-width stream
    for scoring, each as GB/s of the bytes it must move (fixed-width codes,
    encoded blocks, float32 rows) against the HBM peak."""
    ctx.profile_reset()
    ctx.profile_only("store_block_encode,store_block_pack,store_block_decode,store_block_expand")
    ctx.profile(True)
    xhat = torch.empty((store.size, D), dtype=torch.float32, device="cuda")
    for _ in range(reps):
        st = store.block_encode()
        store.block_decode(out=xhat)
    q = torch.zeros((1, D), dtype=torch.float32, device="cuda")
    for _ in range(reps):
        store.score_topk_blocks(q, 1)
    torch.cuda.synchronize()
    ctx.profile(False)
    ctx.profile_only(None)
    n = store.size * D
    fixed = n * st["plain_bits"] / 8
    enc = st["total_bytes"]
    res = {"bits_per_code": st["bits_per_code"], "plain_bits": st["plain_bits"]}
    moved = {"store_block_encode": fixed, "store_block_pack": fixed + enc, "store_block_decode": enc + 4 * n,
             "store_block_expand": enc + fixed}
    for name, b in moved.items():
        tot, cnt = ctx.profile_read(name)
        if cnt:
            gbs = b / (tot / cnt / 1e3) / 1e9
            res[name] = {"us_per_launch": tot / cnt * 1e3, "GBps": gbs, "frac_of_spec": gbs / HBM_PEAK_GBS}
    del xhat
    return res


def band_grid(lam, torch, np, synth, ctx):
    """Band width x quantizer step grid (Appendix "Band width and quantizer
    step") on the subset stream: per setting the candidate share of the
    exhaustive pairs, removal recall against exhaustive greedy and the
    stream's ingest time."""
    cfg = synth.subset_ingest()
    xfull = torch.from_numpy(cfg["x"]).cuda()

    def exhaustive(xd):
        n = xd.shape[0]
        plain = lam.Store(D, TAU, n, ctx=ctx)
        rep = torch.cat([plain.ingest(xd[b0:b0 + BATCH])[0] for b0 in range(0, n, BATCH)]).cpu().numpy()
        return rep, int(np.concatenate([[0], np.cumsum(rep < 0)[:-1]]).sum())

    # Settings whose candidates exceed a fifth of the exhaustive pairs on the
    # stream's first 4,096 arrivals are reported on that prefix only: there
    # most arrivals overflow the per-arrival candidate set.
    xpre = xfull[:BAND_PREFIX]
    rep_full, pairs_full = exhaustive(xfull)
    rep_pre, pairs_pre = exhaustive(xpre)
    pairs = pairs_full
    grid = []
    for r in (2, 4, 8, 16, 32):
        for rel in (0.01, 0.05, 0.1, 0.2, 0.3):
            pt = banded_ingest(lam, torch, np, xpre, rep_pre, pairs_pre, ctx, r=r, rel=rel, reps=1, screened=False)
            pt["arrivals"] = BAND_PREFIX
            if pt["candidate_frac"] <= 0.2:
                pt = banded_ingest(lam, torch, np, xfull, rep_full, pairs_full, ctx, r=r, rel=rel, reps=2,
                                   screened=False)
                pt["arrivals"] = int(xfull.shape[0])
            grid.append(pt)
            print(json.dumps({"progress": [r, rel], "ms": round(pt["ms_per_stream"], 2),
                              "candidate_frac": round(pt["candidate_frac"], 5),
                              "removal_recall": round(pt["removal_recall"], 4)}), file=sys.stderr, flush=True)
    return {"workload": cfg["name"], "tau": TAU, "sigma": 1.0 / D ** 0.5, "exhaustive_pairs": pairs,
            "exhaustive_removal": float(np.mean(rep_full >= 0)), "grid": grid}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the library has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)
    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    import numpy as np
    import torch
    import synth
    import paper_2609_32256_amd as lam

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.band_grid:
        print(json.dumps(band_grid(lam, torch, np, synth, lam.default_context())), flush=True)
        return

    # ------------------------------------------------------------ inputs (resident in HBM)
    raw = synth.raw_qeps(log2n=RAW_LOG2N)["x"]
    n_raw = raw.size
    raw_sets = [torch.from_numpy(raw).to(dev)]
    for s in range(1, RAW_SETS):   # same values, distinct buffers (cache rotation)
        raw_sets.append(raw_sets[0].clone())
    p_raw = lam.qeps_plan(EPS, 1.0, "bits", n_raw)
    raw_codes = [torch.empty(p_raw.code_bytes // 4, dtype=torch.int32, device=dev) for _ in range(RAW_SETS)]
    raw_out = [torch.empty(n_raw, dtype=torch.float32, device=dev) for _ in range(RAW_SETS)]
    p_wide = lam.qeps_plan(min(QEPS_WIDTH_EPS), 1.0, "bits", n_raw)   # the widest codes of the width sweep
    width_codes = [] if args.no_extras else [torch.empty(p_wide.code_bytes // 4, dtype=torch.int32, device=dev)
                                             for _ in range(RAW_SETS)]

    cfg = synth.subset_ingest()
    x = cfg["x"]
    xd = torch.from_numpy(x).to(dev)
    qd = torch.from_numpy(cfg["q"]).to(dev)
    n = x.shape[0]
    ctx = lam.default_context()
    store = lam.Store(D, TAU, n, ctx=ctx)
    xhat = torch.empty((n, D), dtype=torch.float32, device=dev)
    topk_out = (torch.empty((qd.shape[0], TOPK), dtype=torch.float32, device=dev),
                torch.empty((qd.shape[0], TOPK), dtype=torch.int64, device=dev),
                torch.empty(qd.shape[0], dtype=torch.float32, device=dev))
    reps = [torch.empty(min(BATCH, n - b0), dtype=torch.int64, device=dev) for b0 in range(0, n, BATCH)]

    # the raw encode does not wait: its invalid-input counters are checked
    # after the timed steps
    qstatus = torch.zeros(2, dtype=torch.int32, device=dev)

    def step(i):
        k = i % RAW_SETS
        _, p = lam.quantize_async(raw_sets[k], EPS, 1.0, qstatus, out=raw_codes[k], ctx=ctx)
        lam.dequantize(raw_codes[k], p, out=raw_out[k], ctx=ctx)
        store.clear()
        for bi, b0 in enumerate(range(0, n, BATCH)):
            store.ingest(xd[b0:b0 + BATCH], rep=reps[bi], sync=False)   # store.quantize waits for them
        store.quantize(EPS)
        store.dequantize(out=xhat)
        store.score_topk(qd, TOPK, out=topk_out)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # algorithmic pair counts from the decisions (identical every step)
    rep = torch.cat(reps).cpu().numpy()
    kept = rep < 0
    kept_before = np.concatenate([[0], np.cumsum(kept)[:-1]])
    pairs = int(kept_before.sum())                       # sum over arrivals of |R| at arrival
    screen_store_pairs = 0
    screen_chunk_pairs = 0
    for b0 in range(0, n, BATCH):
        nb = min(BATCH, n - b0)
        screen_store_pairs += nb * int(kept_before[b0])
        screen_chunk_pairs += nb * (nb - 1) // 2
    n_store = int(kept.sum())
    info = store.info()

    # 1. instrumented pass: HIP events around every launch, for the per-kernel
    #    breakdown (the events cost time of their own, so this pass is not timed)
    prof_steps = max(2, min(args.steps, 10))
    ctx.profile_reset()
    ctx.profile_only(None)
    ctx.profile(True)
    for i in range(prof_steps):
        step(args.warmup + i)
    torch.cuda.synchronize()
    ctx.profile(False)
    kinfo = {}
    for name in KERNELS:
        tot, cnt = ctx.profile_read(name)
        if cnt:
            kinfo[name] = {"ms_per_step": tot / prof_steps, "launches_per_step": cnt / prof_steps,
                           "avg_launch_ms": tot / cnt}
    dominant = max(kinfo, key=lambda k: kinfo[k]["ms_per_step"])

    # 2. timed pass: events carried by the launches of the dominant kernel and
    #    of the raw Q_eps encode / decode (no marker packets between launches)
    ctx.profile_reset()
    ctx.profile_only(f"{dominant},qeps_encode,qeps_decode")
    ctx.profile(True)
    torch.cuda.synchronize()
    # events between the steps on the library's stream (torch's current one)
    # give the spread of the step time without a synchronisation per step
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t0 = time.perf_counter()
    evs[0].record()
    for i in range(args.steps):
        step(args.warmup + prof_steps + i)
        evs[i + 1].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    step_ms = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
    ctx.profile(False)
    ctx.profile_only(None)
    ms = (t1 - t0) * 1e3 / args.steps
    dom_tot, dom_cnt = ctx.profile_read(dominant)
    timed_qeps = {name: ctx.profile_read(name) for name in ("qeps_encode", "qeps_decode")}
    if qstatus.any().item():
        print(f"raw Q_eps input reported invalid: {qstatus.tolist()}", file=sys.stderr)
        sys.exit(1)

    if args.copy_calibration:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    bq = p_raw.bits / 8.0
    store_elems = n_store * D
    bs = info.q.bits / 8.0
    screen_bytes = 2.0 * D * (screen_store_pairs / BATCH + n) + 8.0 * n   # fp16 store + chunk rows, norms
    work = {  # algorithmic units per step: (amount, unit, peak, bound, algorithmic bytes)
        "qeps_encode": ((4 + bq) * n_raw / 1e9, "GB", HBM_PEAK_GBS, "hbm", (4 + bq) * n_raw),
        "qeps_decode": ((4 + bq) * n_raw / 1e9, "GB", HBM_PEAK_GBS, "hbm", (4 + bq) * n_raw),
        "store_encode": ((4 + bs) * store_elems / 1e9, "GB", HBM_PEAK_GBS, "hbm", (4 + bs) * store_elems),
        "store_decode": ((4 + bs) * store_elems / 1e9, "GB", HBM_PEAK_GBS, "hbm", (4 + bs) * store_elems),
        "dedup_screen": (2.0 * D * (screen_store_pairs + screen_chunk_pairs) / 1e12, "TFLOP",
                         MFMA_F16_PEAK_TFLOPS, "mfma", screen_bytes),
        "score_mfma": (2.0 * D * qd.shape[0] * n_store / 1e12, "TFLOP", MFMA_F16_PEAK_TFLOPS, "mfma", None),
    }
    for name, (amt, unit, peak, bound, _) in work.items():
        if name in kinfo:
            rate = amt / (kinfo[name]["ms_per_step"] / 1e3)
            kinfo[name].update({"achieved": rate, "unit": unit + "/s", "peak": peak, "frac": rate / peak})
    # the raw Q_eps kernels as timed by their own launches in the timed steps
    qeps_timed = {}
    for name, (tot, cnt) in timed_qeps.items():
        if cnt:
            gbs = work[name][0] / (tot / cnt / 1e3)
            qeps_timed[name] = {"us_per_launch": tot / cnt * 1e3, "GBps": gbs, "frac_of_spec": gbs / HBM_PEAK_GBS}
    dom_work = work.get(dominant)
    if dom_work and dom_cnt:
        launches = dom_cnt / args.steps
        per_launch = dom_work[0] / launches
        avg_s = dom_tot / dom_cnt / 1e3
        achieved = per_launch / avg_s
        roofline = {"kernel": dominant, "bound": dom_work[3], "achieved": achieved,
                    "peak": dom_work[2], "unit": "GB/s" if dom_work[1] == "GB" else "TFLOP/s",
                    "frac": achieved / dom_work[2], "traffic": measured_traffic(dominant),
                    "avg_launch_us": avg_s * 1e6, "launches_per_step": launches,
                    "algorithmic_per_launch": per_launch * (1e3 if dom_work[1] == "GB" else 1.0),
                    "algorithmic_unit": "MB" if dom_work[1] == "GB" else "TFLOP",
                    "algorithmic_bytes_per_launch": (dom_work[4] / launches if dom_work[4] else None),
                    "counts": ("screened pairs: each call's rows against the rows retained before it, plus the "
                               "call's lower triangle, 2 D flop each" if dominant == "dedup_screen" else
                               "algorithmic units of the kernel")}
    else:
        roofline = {"kernel": dominant, "bound": "latency", "achieved": None, "peak": None, "unit": None,
                    "frac": None, "traffic": None}

    extras = {}
    if not args.no_extras:
        extras = beside_the_step(lam, torch, np, xd, qd, store, rep, pairs, ctx, raw_sets, raw_out, width_codes)
        tgbs = extras["triad"]["GBps"]
        for v in qeps_timed.values():
            v["frac_of_triad"] = v["GBps"] / tgbs
        if roofline.get("bound") == "mfma" and roofline.get("achieved"):
            roofline["frac_of_matmul_anchor"] = roofline["achieved"] / extras["matmul_anchor"]["TFLOPs"]

    value = pairs / (ms / 1e3) / 1e6
    out = {
        "metric": "Q_eps encode GB/s; near-dup M pairs/s at D=768; queries/s; % of roofline",
        "value": value,
        "unit": "M pairs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "step_ms_p50": float(np.percentile(step_ms, 50)),
        "step_ms_p90": float(np.percentile(step_ms, 90)),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {
            "workload": (f"subset ingest: {n} x {D} float32 unit rows in 600 trajectories, batches of {BATCH}, "
                         f"tau={TAU}; store Q_eps eps={EPS} + decode; {qd.shape[0]} queries top-{TOPK}; "
                         f"plus raw Q_eps encode+decode of 2^{RAW_LOG2N} float32 at eps={EPS}"),
            "pairs_per_step": pairs,
            "screened_pairs_per_step": screen_store_pairs + screen_chunk_pairs,
            "retained": n_store,
            "store_code_bits": int(info.q.bits),
            "raw_code_bits": int(p_raw.bits),
        },
        "qeps_encode_GBps": qeps_timed.get("qeps_encode", {}).get("GBps"),
        "qeps_timed": qeps_timed,
        # every scoring launch: prep, sample, filter, select and rescore, fallback
        "queries_per_s": (qd.shape[0] / (sum(kinfo[k]["ms_per_step"] for k in KERNELS
                                             if k.startswith("score_") and k in kinfo) / 1e3)),
        "roofline": roofline,
        **extras,
        "kernels": kinfo,
        "kernels_note": (f"per-kernel breakdown from {prof_steps} separate steps with HIP events around every "
                         f"launch; the timed steps carry events on the dominant kernel only"),
    }
    if not args.no_cpu_baseline:
        ref, cb = cpu_baseline(x, pairs, raw, cfg["q"])
        if not np.array_equal(ref["rep"], rep):
            raise SystemExit("GPU decisions differ from the oracle on the benchmark stream")
        out["cpu_baseline"] = cb
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
