#!/usr/bin/env python3
"""Throughput of the token-aware verifier hot path on one MI355X.

A step is one pass of the whole offline path over one batch: per-token
features of every logit row (pr_token_features), per-request summaries and
score (pr_request_aggregate) and the ship decision (pr_route). The default
workload is the ragged batch of 64 requests with lengths U{16..512}
(about 16.9k rows) of V = 151,936 bfloat16 logits at T = 0.7; inputs are
generated on the GPU before timing and stay resident in HBM.

Prints one JSON line: rows/s (value), the row kernel's achieved HBM GB/s
against the 8 TB/s peak (roofline, from HIP events around each launch in
the timed region) and the fp64 oracle's rows/s on the host (cpu_baseline,
a bounded sample), plus a parity spot check of that sample. Before the
warmup steps the device is brought to steady clocks by 0.15 s of read-probe
launches (spin_up in the line), since the first launches after an idle
spell run up to 50 % slow.
"""

from __future__ import annotations

import argparse
import gc
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBS = 8000.0


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="ragged_64req_v151936_bf16")
    ap.add_argument("--path", choices=("features", "sample", "sequence", "pipeline", "calibrate"), default="features",
                    help="features: per-token features, per-request summaries and route (the default); "
                         "sequence: the paper's verifier input sequence (l, m, top-20 entropy, t/T) per token; "
                         "pipeline: that sequence, the paper's transformer head (synthetic weights) and route; "
                         "sample: each row's token drawn in the same pass as its features (fused "
                         "sample-and-verify), then summaries and route; "
                         "calibrate: the threshold for a ship fraction on a validation pool of --pool scores")
    ap.add_argument("--pool", type=int, default=8192, help="validation pool size of --path calibrate")
    ap.add_argument("--ship-fraction", type=float, default=0.7, help="ship fraction of --path calibrate")
    ap.add_argument("--stream-quantile", choices=("exact", "p2"), default="exact",
                    help="streaming workloads: exact tail quantile from a per-token history, or the "
                         "bounded-memory P-square estimate")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="time budget of the oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also time a plain device copy of known size (HBM counter calibration)")
    ap.add_argument("--traffic-json", default=os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                                           "profiles", "traffic.json"))
    return ap.parse_args()


def log(msg):
    print(msg, file=sys.stderr, flush=True)


MFMA_F32_PEAK_TFLOPS = 157.3  # dense float32 matrix/vector peak of the part


def head_flops(lengths) -> float:
    """Floating-point operations of the verifier head over requests of these
    lengths: per token the 4 -> 64 projection, per layer the QKV, output and
    feed-forward products and the attention products (QK^T, PV) over the
    request's tokens."""
    T = np.asarray(lengths, dtype=np.float64)
    per_layer = 2 * T * 64 * 192 + 2 * 2 * T * T * 64 + 2 * T * 64 * 64 + 2 * 2 * T * 64 * 128
    return float(np.sum(2 * T * 4 * 64 + 2 * per_layer))


def algorithmic_bytes_per_row(V: int, elem_bytes: int) -> int:
    # one read of the logit row + sampled id and temperature in + 10 outputs of 4 bytes
    return V * elem_bytes + 4 + 4 + 10 * 4


def copy_probe(torch, nbytes=1 << 30, reps=10):
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    return {"bytes_read": nbytes, "bytes_written": nbytes, "ms": ms, "gb_per_s": 2 * nbytes / ms / 1e6}


# ---------------------------------------------------------------------------
# The fp64 oracle on the host's cores (a baseline, not the target)

_ORACLE_DATA = {}


def _oracle_init(path, dtype, mode, top_k):
    """Worker set-up: the sample rows, memory-mapped from the files the parent wrote."""
    import oracle  # noqa: F401  (imported once per worker, outside the timed tasks)
    _ORACLE_DATA.update({k: np.load(os.path.join(path, f"{k}.npy"), mmap_mode="r")
                         for k in ("raw", "ids", "T", "P", "rho") if os.path.exists(os.path.join(path, f"{k}.npy"))})
    _ORACLE_DATA.update(dtype=dtype, mode=mode, top_k=top_k)


def _oracle_rows(rows):
    """The oracle on some rows of the sample: per-token features (mode
    "features") or the verifier input tuple (mode "sequence")."""
    import oracle
    from oracle import sequence as oseq
    d = _ORACLE_DATA
    out = []
    for r in rows:
        raw = np.asarray(d["raw"][r])
        P = None if "P" not in d else float(d["P"][r])
        f = oracle.token_features(raw, d["dtype"], int(d["ids"][r]), float(d["T"][r]), P)
        if d["mode"] == "sequence":
            h = -oseq.topk_entropy(raw, d["dtype"], float(d["T"][r]), P, d["top_k"])
            f = (f["logprob"], f["maxprob"], h, float(d["rho"][r]))
        out.append(f)
    return out


def _noop(_):
    return os.getpid()


def host_cores() -> int:
    """Usable host cores: the affinity mask, capped at the 16 that one GPU's share holds."""
    return max(1, min(len(os.sched_getaffinity(0)), 16))


def cpu_baseline(torch, batch, gpu_out, seconds, mode="features", top_k=20, skip=()):
    """The unchanged fp64 oracle on the first rows of the batch, timed on the
    host: first on one core, then row-parallel over every usable core (a
    process per core, rows handed out four at a time). Every row it computed
    is compared with the GPU's output, and the whole requests among them are
    summarised, scored and routed by the oracle. Time-bounded by `seconds`."""
    import multiprocessing as mp
    import shutil
    import tempfile
    from paper_2608_28726_amd import workloads as wl
    from oracle import aggregate as oagg
    from oracle import sequence as oseq
    w = batch.workload
    dtype = "bf16" if w.dtype == "bf16" else "f32"
    cores = host_cores()
    n_max = min(batch.n_rows, int(3e9 // (w.V * w.elem_bytes)), 8192)
    tmp = tempfile.mkdtemp(prefix="prouter_oracle_", dir="/dev/shm" if os.path.isdir("/dev/shm") else None)
    try:
        np.save(os.path.join(tmp, "raw.npy"), wl.to_host_raw(batch.logits[:n_max]))
        np.save(os.path.join(tmp, "ids.npy"), batch.sampled_ids[:n_max].cpu().numpy())
        np.save(os.path.join(tmp, "T.npy"), batch.temperature[:n_max].cpu().numpy())
        if batch.top_p is not None:
            np.save(os.path.join(tmp, "P.npy"), batch.top_p[:n_max].cpu().numpy())
        if mode == "sequence":
            np.save(os.path.join(tmp, "rho.npy"), oseq.position_fraction(batch.offsets)[:n_max])
        # one core, in this process
        _oracle_init(tmp, dtype, mode, top_k)
        res = []
        t0 = time.perf_counter()
        n1_cap = max(8, n_max // 4)  # leave rows for the all-core run on small batches
        while len(res) < min(n_max, 8) or (len(res) < n1_cap and time.perf_counter() - t0 < 0.3 * seconds):
            res += _oracle_rows([len(res)])
        t1 = time.perf_counter() - t0
        n1 = len(res)
        rate1 = n1 / t1
        # every usable core, a process each (spawned: no GPU state is inherited)
        m = max(0, min(n_max - n1, int(rate1 * cores * 0.7 * seconds)))
        ctx = mp.get_context("spawn")
        with ctx.Pool(cores, initializer=_oracle_init, initargs=(tmp, dtype, mode, top_k)) as pool:
            pool.map(_noop, range(4 * cores))  # workers up and the oracle imported
            tasks = [list(range(a, min(n1 + m, a + 4))) for a in range(n1, n1 + m, 4)]
            t0 = time.perf_counter()
            parts = pool.map(_oracle_rows, tasks, chunksize=1)
            tN = time.perf_counter() - t0
        for part in parts:
            res += part
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    n = len(res)
    rateN = m / tN if m else rate1
    # parity of every computed row against the GPU's outputs
    bad, detail = 0, {}
    if mode == "sequence":
        Xo = np.array(res, dtype=np.float64)
        Xg = gpu_out[:n].cpu().numpy().astype(np.float64)
        with np.errstate(invalid="ignore"):
            ok = (np.abs(Xg - Xo) <= 1e-5 + 1e-4 * np.abs(Xo)) | (np.isnan(Xg) & np.isnan(Xo)) | (Xg == Xo)
        bad = int((~ok).sum())
        if bad:
            i = np.argwhere(~ok)[:3].tolist()
            detail["X"] = {"count": bad, "at": i}
        what = f"the verifier input tuple (log-prob, max-prob, top-{top_k} entropy, position fraction)"
        n_whole = 0
    else:
        amb = np.array([d["ambiguous"] for d in res])
        for k in ("max_logit", "lse", "entropy", "logprob", "maxprob", "margin", "rank", "argmax", "cutoff", "flags"):
            if k in skip:
                continue
            g = gpu_out[k][:n].cpu().numpy()
            o = np.array([d[k] for d in res])
            if k in ("rank", "argmax", "cutoff", "flags"):
                g = g.astype(np.int64) & 0xFFFFFFFF if k == "flags" else g
                bad_k = (g != o) & ~(amb if k in ("cutoff", "flags") else np.zeros(n, bool))
            else:
                g = g.astype(np.float64)
                with np.errstate(invalid="ignore"):
                    ok = (np.abs(g - o) <= 1e-5 + 1e-4 * np.abs(o)) | (np.isnan(g) & np.isnan(o)) | (g == o)
                bad_k = ~ok & ~(amb if k in ("lse", "entropy", "logprob", "maxprob") else np.zeros(n, bool))
            bad += int(bad_k.sum())
            if bad_k.any():
                i = np.flatnonzero(bad_k)[:3]
                detail[k] = {"count": int(bad_k.sum()), "rows": i.tolist(), "gpu": g[i].tolist(), "oracle": o[i].tolist()}
        # whole requests inside the sample: summaries, score and route
        offs = batch.offsets
        n_whole = int(np.searchsorted(offs, n, side="right")) - 1
        if n_whole > 0:
            of = {k: np.array([d[k] for d in res]) for k in ("logprob", "maxprob", "entropy", "margin")}
            oagg.route(oagg.score_from_aggregates(oagg.request_aggregate(of, offs[: n_whole + 1], q=w.q)), w.tau)
        what = "all per-token features"
    if detail:
        log(f"[bench] parity detail: {json.dumps(detail)}")
    return {
        "value": rateN,
        "unit": "rows/s",
        "cores": cores,
        "kind": "oracle",
        "sample": f"first {n} rows ({n_whole} whole requests) of the same batch: {what} in float64 "
                  f"(numpy, one process per core); {n1} rows on 1 core in {t1:.1f} s, then {m} rows on "
                  f"{cores} cores in {tN:.1f} s" if m else f"first {n} rows on 1 core in {t1:.1f} s",
        "single_core": {"value": rate1, "unit": "rows/s", "cores": 1, "rows": n1, "seconds": t1},
        "parity_mismatches": bad,
        "rows": n,
    }


def read_probe(torch, wl, buffers, reps=4):
    """Practical read ceiling, measured in this run: the plain read-only probe
    (nontemporal 16-byte loads, nothing computed) over the same resident
    inputs, cycling through `buffers` (tensors); the best of a few grid sizes."""
    import ctypes
    L = wl.tools()
    stream = torch.cuda.current_stream()
    best = None
    shapes = ((4096, 8, 256), (8192, 8, 256), (16384, 4, 256), (16384, 8, 256), (8192, 8, 512), (16384, 4, 512),
              (16384, 8, 512), (8192, 8, 1024), (16384, 8, 1024), (16384, 16, 1024))
    for blocks, unroll, threads in shapes:
        sink = torch.zeros(blocks * threads, dtype=torch.int32, device="cuda")
        nb = [(b.numel() * b.element_size()) // 16 * 16 for b in buffers]

        def launch(k):
            st = L.prt_read_probe(ctypes.c_void_p(buffers[k % len(buffers)].data_ptr()), nb[k % len(buffers)],
                                  ctypes.c_void_p(sink.data_ptr()), blocks, unroll, threads,
                                  ctypes.c_void_p(stream.cuda_stream))
            if st != 0:
                raise RuntimeError(f"prt_read_probe failed with status {st}")
        launch(0)
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(reps * len(buffers))]
        for k, (a, b) in enumerate(ev):
            a.record()
            launch(k + 1)
            b.record()
        torch.cuda.synchronize()
        ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
        nbytes = float(np.mean(nb))
        gbs = nbytes / (ms * 1e-3) / 1e9
        if best is None or gbs > best["gb_per_s"]:
            best = {"gb_per_s": gbs, "bytes_per_launch": nbytes, "ms": ms, "blocks": blocks,
                    "threads_per_workgroup": threads, "loads_in_flight_per_thread": unroll,
                    "kernel": f"read_probe_kernel (nontemporal 16-byte loads; best of {len(shapes)} launch shapes)"}
    return best


def spin_up(torch, wl, buffers, seconds=0.15):
    """Brings the device to its steady clocks before anything is timed. After
    an idle spell the first launches run slow (the row kernel took 1.05-1.25
    ms instead of 0.81 for its first launches after 2 s idle, and about 30
    launches to settle), which a few warmup steps do not cover. This reads
    the resident inputs with the plain read probe (one launch shape, nothing
    computed, nothing kept) for `seconds` of wall time; it precedes the
    warmup steps and is not part of any timed region."""
    import ctypes
    L = wl.tools()
    stream = torch.cuda.current_stream()
    blocks, unroll, threads = 16384, 8, 512
    sink = torch.zeros(blocks * threads, dtype=torch.int32, device="cuda")
    nb = [(b.numel() * b.element_size()) // 16 * 16 for b in buffers]
    launches, t0 = 0, time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(8):
            k = launches % len(buffers)
            st = L.prt_read_probe(ctypes.c_void_p(buffers[k].data_ptr()), nb[k], ctypes.c_void_p(sink.data_ptr()),
                                  blocks, unroll, threads, ctypes.c_void_p(stream.cuda_stream))
            if st != 0:
                raise RuntimeError(f"prt_read_probe failed with status {st}")
            launches += 1
        torch.cuda.synchronize()
    return {"seconds": time.perf_counter() - t0, "launches": launches,
            "kernel": "read_probe_kernel over the resident inputs, before the warmup steps (untimed)"}


def run_offline(args, torch, pr, wl, w):
    """Offline ragged batches (features -> summaries -> route per step). Workloads
    larger than one batch are generated as device-resident chunks of whole
    requests; small ones are replicated so that a step never re-reads the
    256 MB last-level cache."""
    n_chunks = 16 if w.n_req * w.len_hi * w.V * w.elem_bytes > 40e9 else 1
    per = w.n_req // n_chunks
    batches = [wl.make_batch(wl.scaled(w, n_req=per, seed=w.seed + c) if n_chunks > 1 else w, device="cuda")
               for c in range(n_chunks)]
    copies = 1
    one = batches[0].n_rows * w.V * w.elem_bytes
    if n_chunks == 1 and one < 512e6:
        copies = int(np.ceil(600e6 / one))
        base = batches[0]
        batches = [base] + [wl.Batch(base.workload, base.offsets, base.logits.clone(), base.sampled_ids,
                                     base.temperature, base.top_p) for _ in range(copies - 1)]
    torch.cuda.synchronize()
    n_rows = sum(b.n_rows for b in batches) // copies
    log(f"[bench] {w.name}: {n_rows} rows in {n_chunks} chunk(s), {copies} rotating copies, "
        f"{n_rows * w.V * w.elem_bytes / 1e9:.2f} GB per step")
    offs = [torch.as_tensor(b.offsets).cuda() for b in batches]
    sequence = args.path in ("sequence", "pipeline")
    pipeline = args.path == "pipeline"
    sample = args.path == "sample"
    drawn = [torch.empty(b.n_rows, dtype=torch.int32, device="cuda") for b in batches] if sample else None
    if pipeline:
        head_w = torch.tensor(wl.head_weights(), device="cuda")
        head_ws = [torch.empty(max(int(pr._abi.lib().pr_verifier_head_workspace(b.n_rows)), 1), dtype=torch.uint8,
                               device="cuda") for b in batches]
        head_ev = []
    if sequence:
        feats = [torch.empty(b.n_rows, 4, dtype=torch.float32, device="cuda") for b in batches]
    else:
        feats = [pr.token_features(b.logits, b.sampled_ids, b.temperature, b.top_p) for b in batches]
    wss = []
    for b in batches:
        nb = 0 if sequence else pr.token_features_workspace(b.logits, b.top_p is not None)
        wss.append(torch.empty(max(nb, 1), dtype=torch.uint8, device="cuda"))
    state = {"k": 0}

    def step(ev=None):
        group = [state["k"] % copies] if copies > 1 else range(n_chunks)
        state["k"] += 1
        out = None
        for c in group:
            b = batches[c]
            if ev is not None and c == group[0]:
                ev[0].record()
            if sequence:
                pr.feature_sequence(b.logits, b.sampled_ids, b.temperature, offs[c], top_p=b.top_p,
                                    top_k=pr.PAPER_TOP_K, out=feats[c])
            elif sample:
                pr.sample_features(b.logits, b.temperature, seed=20261202, offset=state["k"], ids_out=drawn[c],
                                   out=feats[c])
            else:
                pr.token_features(b.logits, b.sampled_ids, b.temperature, b.top_p, out=feats[c],
                                  workspace=wss[c])
            if ev is not None and c == group[-1]:
                ev[1].record()
            if pipeline:
                h0, h1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                h0.record()
                scores = pr.verifier_head(feats[c], offs[c], head_w, max_len=w.len_hi, workspace=head_ws[c])
                h1.record()
                if ev is not None:
                    head_ev.append((h0, h1))
                out = pr.route(scores, w.tau)
            elif not sequence:
                agg = pr.request_aggregate(feats[c], offs[c], q=w.q)
                out = pr.route(agg["score"], w.tau)
        return out

    # The collector stays off from before the spin-up to the end of the timed
    # region: a collection pass in the timed region once held back a launch by
    # 1.2 ms, and one between the warm-up and the timed steps idles the device.
    gc.collect()
    gc.disable()
    spun = spin_up(torch, wl, [b.logits for b in batches[:max(1, copies)]])
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    events = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    log(f"[bench] timing {args.steps} steps")
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(events[k])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    gc.enable()
    kern_times = [a.elapsed_time(b) for a, b in events]
    kern_ms = float(np.mean(kern_times))
    if sequence:  # one read of the row, id and temperature in, the 16-byte tuple out
        bytes_launch = n_rows * (w.V * w.elem_bytes + 4 + 4 + 16)
    else:
        bytes_launch = n_rows * algorithmic_bytes_per_row(w.V, w.elem_bytes)
    kernel = "topp_kernel" if w.P_lo is not None else "row_features_kernel"
    if sequence:
        kernel += " (sequence variant)"
    if sample:
        kernel += " (sampling variant)"
    if n_chunks > 1:  # events bracket all chunks' row kernels and their summaries
        kernel += f" x{n_chunks} chunks (+summaries)"
    extra = {"kernel": kernel, "kernel_ms": kern_ms, "kernel_ms_median": float(np.median(kern_times)),
             "kernel_ms_per_step": [round(float(x), 4) for x in kern_times],
             "timing": f"kernel_ms: mean over the {args.steps} timed steps of HIP events recorded around the "
                       "launch on its stream; achieved = bytes_per_launch / kernel_ms",
             "bytes_per_launch": bytes_launch,
             "_probe_buffers": [b.logits for b in batches[:max(1, copies)]], "_spin_up": spun}
    if pipeline:
        head_ms = float(np.mean([a.elapsed_time(b) for a, b in head_ev]))
        flops = sum(head_flops(np.diff(b.offsets)) for b in batches) / copies
        extra["head"] = {"ms": head_ms, "gflop": flops / 1e9, "tflop_per_s": flops / (head_ms * 1e-3) / 1e12,
                         "peak_tflop_per_s": MFMA_F32_PEAK_TFLOPS, "weights": "synthetic (seeded)"}
        log(f"[bench] verifier head {head_ms * 1e3:.1f} us per batch, {flops / 1e9:.2f} GFLOP")
    if sample:  # the oracle baseline checks the drawn rows' features for the drawn ids
        b = batches[0]
        pr.sample_features(b.logits, b.temperature, seed=20261202, offset=0, ids_out=drawn[0], out=feats[0])
        torch.cuda.synchronize()
        return (wl.Batch(b.workload, b.offsets, b.logits, drawn[0], b.temperature, b.top_p), feats[0], n_rows,
                elapsed, kern_ms, bytes_launch, extra)
    return batches[0], feats[0], n_rows, elapsed, kern_ms, bytes_launch, extra


def run_stream(args, torch, pr, wl, w):
    """Streaming decode: one pr_stream_step per decode step over the active
    slots, pr_stream_finish for the slots whose request ends. The whole
    schedule of 1,024 steps is one pass; it is captured once in a HIP graph
    and replayed, so that the timed region holds the GPU work of the pass
    without the host's per-call overhead. Every replay's verdicts are
    checked against an eager pass. The row kernel's time per full step (256
    rows) comes from a graph of back-to-back full steps."""
    fin = wl.stream_schedule(w)
    n_steps = int(fin.max())
    pool = []
    for p in range(6):  # 6 x 78 MB of distinct step inputs, cycled (above the 256 MB cache)
        pool.append(wl.stream_step_inputs(w, 10_000 + p, np.arange(w.n_req), device="cuda"))
    torch.cuda.synchronize()
    st = pr.StreamState(w.n_req, n_steps if args.stream_quantile == "exact" else 0, q=w.q)
    actives = [torch.as_tensor(np.flatnonzero(fin >= s).astype(np.int32), device="cuda") for s in range(1, n_steps + 1)]
    endings = [torch.as_tensor(np.flatnonzero(fin == s).astype(np.int32), device="cuda") for s in range(1, n_steps + 1)]
    rows = int(sum(a.shape[0] for a in actives))

    def one_pass(events=None):
        outs = []
        for s in range(n_steps):
            act = actives[s]
            n = act.shape[0]
            logits, ids, T = pool[s % len(pool)]
            if events is not None:
                events[s][0].record()
            st.step(logits[:n], act, ids[:n], T[:n])
            if events is not None:
                events[s][1].record()
            if endings[s].shape[0]:
                outs.append(st.finish(endings[s], w.tau))
        return outs

    def verdicts(outs):
        return [(o["score"].clone(), o["ship"].clone()) for o in outs]

    def same(a, b):
        return all(torch.equal(x[0].view(torch.int32), y[0].view(torch.int32)) and torch.equal(x[1], y[1])
                   for x, y in zip(a, b)) and len(a) == len(b)

    ref = verdicts(one_pass())  # eager pass (also clears every slot at its finish)
    # Host-paced eager pass with events around each step (per-step latency as a caller sees it).
    events = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n_steps)]
    gc.collect()
    gc.disable()
    t0 = time.perf_counter()
    eager = verdicts(one_pass(events))
    torch.cuda.synchronize()
    eager_s = time.perf_counter() - t0
    gc.enable()
    ks = np.array([a.elapsed_time(b) for a, b in events])
    eager_ok = same(eager, ref)

    # The whole schedule as one graph.
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        one_pass()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        g_outs = one_pass()
    replays_ok = True
    gc.collect()
    gc.disable()
    spun = spin_up(torch, wl, [p[0] for p in pool])
    for _ in range(max(1, args.warmup)):
        g.replay()
        torch.cuda.synchronize()
        replays_ok &= same(verdicts(g_outs), ref)
    reps = max(1, args.steps // 50)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / reps
    gc.enable()
    pass_ms = e0.elapsed_time(e1) / reps
    replays_ok &= same(verdicts(g_outs), ref)

    # Row kernel time per full step: 20 back-to-back full steps in a graph.
    full = torch.arange(w.n_req, dtype=torch.int32, device="cuda")
    n_full = 20
    g2 = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        for k in range(3):
            logits, ids, T = pool[k % len(pool)]
            st.step(logits, full, ids, T)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g2):
        for k in range(n_full):
            logits, ids, T = pool[k % len(pool)]
            st.step(logits, full, ids, T)
    g2.replay()
    torch.cuda.synchronize()
    f0, f1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    f0.record()
    for _ in range(5):
        g2.replay()
    f1.record()
    torch.cuda.synchronize()
    kern_full = f0.elapsed_time(f1) / (5 * n_full)
    st.reset(full)
    st.close()
    if not (eager_ok and replays_ok):
        raise RuntimeError("streaming verdicts of the graph replays differ from the eager pass")

    # The oracle baseline takes the first pool step's rows (one full step of
    # 256 rows), with their features from the same row kernel tier.
    logits0, ids0, T0 = pool[0]
    feats0 = pr.token_features(logits0, ids0, T0)
    torch.cuda.synchronize()
    batch0 = wl.Batch(w, np.array([0, w.n_req], dtype=np.int32), logits0, ids0, T0, None)
    bytes_step = w.n_req * algorithmic_bytes_per_row(w.V, w.elem_bytes)
    extra = {"kernel": "row_features_kernel (streaming step, 256 rows)", "kernel_ms": kern_full,
             "timing": f"kernel_ms: HIP events around {5 * n_full} back-to-back full 256-row steps replayed "
                       "from a graph, divided by their number; achieved = bytes_per_launch / kernel_ms",
             "bytes_per_launch": bytes_step, "_probe_buffers": [p[0] for p in pool], "_spin_up": spun,
             "pass_ms_graph": pass_ms, "wall_ms_graph": wall * 1e3,
             "us_per_step_graph": pass_ms * 1e3 / n_steps,
             "eager_step_us_p50": float(np.percentile(ks, 50) * 1e3),
             "eager_step_us_p99": float(np.percentile(ks, 99) * 1e3),
             "eager_wall_us_per_step": eager_s * 1e6 / n_steps,
             "steps_total": n_steps, "graph_replays_checked": True}
    log(f"[bench] stream: {n_steps} steps, {rows} rows; graph pass {pass_ms:.3f} ms "
        f"({pass_ms * 1e3 / n_steps:.1f} us/step), full-step row kernel {kern_full * 1e3:.1f} us; "
        f"eager (host-paced) p50 {extra['eager_step_us_p50']:.1f} us, wall {extra['eager_wall_us_per_step']:.1f} us/step")
    return batch0, feats0, rows, pass_ms * 1e-3, kern_full, bytes_step, extra


def run_calibrate(args, torch, pr, wl):
    """Threshold calibration on a validation pool (pr_calibrate_threshold):
    one call per step, each bracketed by HIP events on the stream it is
    launched on; the oracle's calibration of the same pool is timed on the
    host and must give the same tau and ship count."""
    import oracle
    n, q = args.pool, args.ship_fraction
    host = wl.validation_scores(n)
    s = torch.from_numpy(host).cuda()
    gc.collect()
    gc.disable()
    for _ in range(max(1, args.warmup)):
        tau, ns = pr.calibrate_threshold(s, q)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    t0 = time.perf_counter()
    for a, b in ev:
        a.record()
        tau, ns = pr.calibrate_threshold(s, q)
        b.record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    gc.enable()
    call_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    c0 = time.perf_counter()
    reps = 0
    while True:
        otau, ons = oracle.calibrate_threshold(host.astype(np.float64), q)
        reps += 1
        if time.perf_counter() - c0 >= min(args.cpu_seconds, 2.0):
            break
    cpu_s = (time.perf_counter() - c0) / reps
    if float(tau.item()) != otau or int(ns.item()) != ons:
        raise RuntimeError(f"calibration differs from the oracle: {tau.item()} {ns.item()} vs {otau} {ons}")
    achieved = 4.0 * n / (call_ms * 1e-3) / 1e9
    result = {
        "metric": "threshold calibrations/sec on a validation pool",
        "value": args.steps / elapsed, "unit": "calibrations/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": elapsed * 1e3 / args.steps, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"validation pool of {n} scores ~ Beta(5,2), 0.5% NaN", "pool": n,
                   "ship_fraction": q},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None, "kernel": "calibrate_kernel",
                     "kernel_ms": call_ms, "bytes_per_launch": 4 * n},
        "cpu_baseline": {"value": 1.0 / cpu_s, "unit": "calibrations/s", "cores": 1, "kind": "oracle",
                         "sample": f"the same pool, {reps} calibrations"},
        "tau": float(tau.item()), "n_ship": int(ns.item()),
    }
    log(f"[bench] calibrate: {n} scores, {call_ms * 1e3:.1f} us per call; oracle {cpu_s * 1e3:.2f} ms")
    print(json.dumps(result), flush=True)


def main():
    args = parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported. Rows and requests are "
              "independent, so several GPUs would each take whole requests with no exchange between them.",
              file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2608_28726_amd as pr
    from paper_2608_28726_amd import workloads as wl
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.path == "calibrate":
        run_calibrate(args, torch, pr, wl)
        return

    w = wl.WORKLOADS[args.workload]
    log(f"[bench] generating {w.name} on the GPU")
    stream_mode = w.name.startswith("stream_")
    runner = run_stream if stream_mode else run_offline
    batch, feats, n_rows, elapsed, avg_ms, bytes_launch, extra = runner(args, torch, pr, wl, w)
    steps = 1 if stream_mode else args.steps
    ms_per_step = elapsed * 1e3 / (int(extra.get("steps_total", 0)) if stream_mode else args.steps)
    rows_per_s = n_rows * (1 if stream_mode else args.steps) / elapsed
    achieved = bytes_launch / (avg_ms * 1e-3) / 1e9
    log(f"[bench] {ms_per_step:.3f} ms/step, row kernel {avg_ms:.3f} ms ({achieved:.0f} GB/s)")

    traffic = stored_traffic(args.traffic_json, w.name, args.path)
    spun = extra.pop("_spin_up")
    probe = read_probe(torch, wl, extra.pop("_probe_buffers"))
    probe["frac_of_probe"] = achieved / probe["gb_per_s"]
    log(f"[bench] read probe {probe['gb_per_s']:.0f} GB/s ({probe['blocks']} workgroups, "
        f"{probe['loads_in_flight_per_thread']} loads in flight); the kernel reaches "
        f"{100 * probe['frac_of_probe']:.1f} % of it")

    result = {
        "metric": "verified token rows/sec and achieved HBM GB/s (% of peak), V=151,936 bf16",
        "value": rows_per_s,
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "n_req": w.n_req, "rows": n_rows, "V": w.V, "logits": w.dtype,
                   "mode": "streaming decode, one step per token" if stream_mode else "offline ragged batch",
                   "path": {"sequence": "verifier input sequence (l, m, top-20 entropy, t/T)",
                            "pipeline": "verifier input sequence, transformer head (synthetic weights), route",
                            "sample": "token drawn in the same pass (fused sample-and-verify), features, "
                                      "summaries, route"}.get(
                                args.path, "features, summaries, route"),
                   "temperature": [w.T_lo, w.T_hi], "top_p": None if w.P_lo is None else [w.P_lo, w.P_hi],
                   "aggregation": (f"mean/min/q={w.q} P-square estimate" if stream_mode and
                                   args.stream_quantile == "p2" else f"mean/min/q={w.q} nearest-rank"),
                   "threshold": w.tau},
        "gb_per_s": achieved,
        "pct_of_hbm_peak": 100.0 * achieved / HBM_PEAK_GBS,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic, **extra},
        "read_probe": probe,
        "spin_up": spun,
    }
    if args.copy_probe:
        result["copy_probe"] = copy_probe(torch)
    if not args.no_cpu_baseline and batch is not None:
        log("[bench] timing the oracle on the host")
        if args.path in ("sequence", "pipeline"):
            result["cpu_baseline"] = cpu_baseline(torch, batch, feats, args.cpu_seconds, mode="sequence",
                                                  top_k=pr.PAPER_TOP_K)
        else:
            result["cpu_baseline"] = cpu_baseline(torch, batch, feats, args.cpu_seconds,
                                                  skip=("rank",) if args.path == "sample" else ())
        log(f"[bench] oracle {result['cpu_baseline']['value']:.1f} rows/s, "
            f"parity mismatches {result['cpu_baseline']['parity_mismatches']}")
    print(json.dumps(result), flush=True)


# Sources each measured kernel is compiled from (its own file and every header it includes).
KERNEL_SOURCES = {
    "row_features_kernel": ("include/prouter.h", "paper_2608_28726_amd/csrc/device_util.h",
                            "paper_2608_28726_amd/csrc/row_features.h", "paper_2608_28726_amd/csrc/row_scan.h",
                            "paper_2608_28726_amd/csrc/topk.h", "paper_2608_28726_amd/csrc/p2.h",
                            "paper_2608_28726_amd/csrc/sample.h", "paper_2608_28726_amd/csrc/row_features.hip"),
    "topp_kernel": ("include/prouter.h", "paper_2608_28726_amd/csrc/device_util.h",
                    "paper_2608_28726_amd/csrc/row_features.h", "paper_2608_28726_amd/csrc/row_scan.h",
                    "paper_2608_28726_amd/csrc/topk.h", "paper_2608_28726_amd/csrc/p2.h",
                    "paper_2608_28726_amd/csrc/topp.h", "paper_2608_28726_amd/csrc/topp.hip"),
}


def traffic_key(workload: str, path: str) -> str:
    """Key of a workload's stored counter traffic (one entry per measured path)."""
    return workload if path == "features" else f"{workload}:{path}"


def stored_traffic(traffic_json: str, workload: str, path: str):
    """HBM bytes per launch from the stored counter runs of this workload and
    path, or None: no record, or one taken on other kernel sources."""
    if not os.path.exists(traffic_json):
        return None
    try:
        t = json.load(open(traffic_json)).get(traffic_key(workload, path))
        if t and t.get("kernel_source_hash") == kernel_source_hash(t.get("kernel", "")):
            return t["bytes_per_launch"]
    except (OSError, ValueError, KeyError):
        pass
    return None


def kernel_source_hash(kernel: str) -> str:
    """Hash of one kernel's sources: stored counter traffic is only valid for the same kernel."""
    import hashlib
    root = os.path.dirname(os.path.abspath(__file__))
    h = hashlib.sha256()
    for fn in KERNEL_SOURCES[kernel]:
        h.update(open(os.path.join(root, fn), "rb").read())
    return h.hexdigest()[:16]


if __name__ == "__main__":
    main()
