"""Writes the expected outputs of the full-size workloads (tests/golden/fullsize_*.npz).

Every value here comes from the float64 oracle (``oracle/``) run on rows made
by the host twin of the seeded logit generator (``workloads.host_rows``); the
sampled ids are drawn by the host sampler (``workloads.host_sample_ids``) and
stored, since the GPU tests read them back as inputs. Nothing here touches
the HIP library. The GPU tests regenerate the same rows on the device, check
their checksums against the stored ones, feed the stored ids and compare
every stored output.

Coverage:
  pr1_ref_8x64_v32000_f32, ragged_64req_v151936_bf16, topp_128x256_v262144_f32:
      every row's features, every request's summaries, score and decision;
  offline_512x512_v151936_bf16: chunks 0 and 15 of the 16 (requests 0-31
      and 480-511, 32,768 rows), every row and request of those chunks;
  stream_256slots_v151936_bf16: the whole 1,024-step schedule: every slot's
      count, summaries, score and decision at its finish, every step's input
      checksum and ids, and every row's features on every 16th step plus the
      first two and the last two.

Usage: python tests/golden/make_fullsize.py [--jobs N] [workload ...]
Runs the oracle row-parallel in N processes (default: all usable cores).
"""

from __future__ import annotations

import argparse
import hashlib
import json
import multiprocessing as mp
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from oracle import aggregate as oagg  # noqa: E402
from paper_2608_28726_amd import workloads as wl  # noqa: E402

FLOATS = ("max_logit", "lse", "entropy", "logprob", "maxprob", "margin")
INTS = ("rank", "argmax", "cutoff")
OFFLINE_CHUNKS_CHECKED = (0, 15)
STREAM_FEATURE_EVERY = 16
ORACLE_FILES = ("oracle/features.py", "oracle/aggregate.py")


def oracle_hash() -> str:
    """Hash of the oracle sources the stored values come from."""
    h = hashlib.sha256()
    for fn in ORACLE_FILES:
        h.update(open(os.path.join(ROOT, fn), "rb").read())
    return h.hexdigest()[:16]


def golden_path(name: str) -> str:
    return os.path.join(HERE, f"fullsize_{name}.npz")


# ---------------------------------------------------------------------------
# Worker side: rows -> (id, checksum, oracle features)

_PLANS: dict = {}


def _plan(w):
    if w.name + str(w.seed) not in _PLANS:
        _PLANS[w.name + str(w.seed)] = wl.batch_plan(w)
    return _PLANS[w.name + str(w.seed)]


def _rows_result(w, raw, seed, row_index, T, P):
    ids = wl.host_sample_ids(raw, T, P, seed, row_index)
    cks = wl.row_checksums(raw)
    f = oracle.token_features_batch(raw, w.dtype, ids, T, P)
    return ids, cks, f


def _batch_task(args):
    w, a, b = args
    offsets, s, h, j, T, P = _plan(w)
    raw = wl.host_rows(w.seed, np.arange(a, b), w.V, w.dtype, s[a:b], h[a:b], j[a:b])
    return a, _rows_result(w, raw, w.seed, np.arange(a, b), T[a:b], None if P is None else P[a:b])


def _stream_task(args):
    w, step, active = args
    idx, s, h, j = wl.stream_rows(w, step, active)
    seed = wl.stream_seed(w)
    raw = wl.host_rows(seed, idx, w.V, w.dtype, s, h, j)
    T = np.full(len(active), np.float32(w.T_lo), dtype=np.float32)
    return step, _rows_result(w, raw, seed, idx, T, None)


# ---------------------------------------------------------------------------
# Parent side

def _concat(parts):
    """Per-row results of consecutive tasks -> ids, checksums, feature arrays."""
    ids = np.concatenate([p[0] for p in parts]).astype(np.int32)
    cks = np.concatenate([p[1] for p in parts]).astype(np.int64)
    f = {k: np.concatenate([p[2][k] for p in parts]) for k in parts[0][2]}
    return ids, cks, f


def _feature_arrays(f, prefix=""):
    out = {}
    for k in FLOATS:
        out[prefix + k] = f[k].astype(np.float64)
    for k in INTS:
        out[prefix + k] = f[k].astype(np.int32)
    out[prefix + "flags"] = f["flags"].astype(np.uint8)
    out[prefix + "ambiguous"] = f["ambiguous"].astype(bool)
    return out


def _request_arrays(f, offsets, w):
    agg = oagg.request_aggregate(f, offsets, q=w.q)
    score = oagg.score_from_aggregates(agg)
    return {"count": agg["count"].astype(np.int32), "mean": agg["mean"], "min": agg["min"], "quant": agg["quant"],
            "score": score, "ship": oagg.route(score, w.tau)}


def _meta(w, extra):
    m = {"workload": w.name, "seed": w.seed, "oracle_hash": oracle_hash(),
         "written": time.strftime("%Y-%m-%d %H:%M:%S"), "generator": "workloads.host_rows (SplitMix64 + quantile table)"}
    m.update(extra)
    return np.frombuffer(json.dumps(m).encode(), dtype=np.uint8)


def batch_golden(w, pool, rows_per_task=32, label=None):
    offsets, s, h, j, T, P = wl.batch_plan(w)
    n = int(offsets[-1])
    tasks = [(w, a, min(n, a + rows_per_task)) for a in range(0, n, rows_per_task)]
    parts = {}
    t0 = time.time()
    for k, (a, res) in enumerate(pool.imap_unordered(_batch_task, tasks)):
        parts[a] = res
        if (k + 1) % max(1, len(tasks) // 20) == 0:
            print(f"  {label or w.name}: {k + 1}/{len(tasks)} tasks, {time.time() - t0:.0f} s", flush=True)
    ids, cks, f = _concat([parts[a] for a in sorted(parts)])
    req_ck = np.array([wl.combine_checksums(cks[offsets[i]:offsets[i + 1]]) for i in range(len(offsets) - 1)],
                      dtype=np.int64)
    out = {"offsets": offsets, "ids": ids, "checksum_req": req_ck, "T": T}
    if P is not None:
        out["P"] = P
    out.update(_feature_arrays(f))
    out.update({"req_" + k: v for k, v in _request_arrays(f, offsets, w).items()})
    out["meta"] = _meta(w, {"n_rows": n, "n_req": len(offsets) - 1, "seconds": time.time() - t0})
    return out


def stream_golden(w, pool):
    fin = wl.stream_schedule(w)
    n_steps = int(fin.max())
    tasks = [(w, step, np.flatnonzero(fin >= step).astype(np.int64)) for step in range(1, n_steps + 1)]
    feature_steps = sorted({1, 2, n_steps - 1, n_steps} | set(range(STREAM_FEATURE_EVERY, n_steps + 1,
                                                                     STREAM_FEATURE_EVERY)))
    per_step = {}
    t0 = time.time()
    for k, (step, res) in enumerate(pool.imap_unordered(_stream_task, tasks)):
        per_step[step] = res
        if (k + 1) % 50 == 0:
            print(f"  {w.name}: {k + 1}/{n_steps} steps, {time.time() - t0:.0f} s", flush=True)
    # slot-major sequences of each slot's rows, in step order
    seqs = {c: {key: [] for key in ("logprob", "maxprob", "entropy", "margin")} for c in range(w.n_req)}
    ids_all, step_off, step_ck = [], [0], []
    feat_parts, feat_off = [], [0]
    for step in range(1, n_steps + 1):
        active = tasks[step - 1][2]
        ids, cks, f = per_step[step]
        ids_all.append(ids)
        step_off.append(step_off[-1] + len(ids))
        step_ck.append(wl.combine_checksums(cks))
        for k, c in enumerate(active):
            for key in seqs[c]:
                seqs[c][key].append(f[key][k])
        if step in feature_steps:
            feat_parts.append(f)
            feat_off.append(feat_off[-1] + len(ids))
    counts = np.array([len(seqs[c]["logprob"]) for c in range(w.n_req)])
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    flat = {key: np.concatenate([np.asarray(seqs[c][key], dtype=np.float64) for c in range(w.n_req)])
            for key in ("logprob", "maxprob", "entropy", "margin")}
    out = {"fin": fin, "ids": np.concatenate(ids_all).astype(np.int32), "step_offsets": np.array(step_off, np.int64),
           "checksum_step": np.array(step_ck, dtype=np.int64), "feature_steps": np.array(feature_steps, np.int32),
           "feature_offsets": np.array(feat_off, np.int64)}
    out.update(_feature_arrays({k: np.concatenate([p[k] for p in feat_parts]) for k in feat_parts[0]}))
    out.update({"slot_" + k: v for k, v in _request_arrays(flat, offsets, w).items()})
    out["meta"] = _meta(w, {"n_steps": n_steps, "rows": int(step_off[-1]), "seconds": time.time() - t0})
    return out


def write(name, arrays):
    path = golden_path(name)
    np.savez_compressed(path, **arrays)
    print(f"wrote {path} ({os.path.getsize(path) / 1e6:.2f} MB)", flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--jobs", type=int, default=len(os.sched_getaffinity(0)))
    ap.add_argument("workloads", nargs="*", default=list(wl.WORKLOADS))
    args = ap.parse_args()
    ctx = mp.get_context("fork")
    with ctx.Pool(args.jobs) as pool:
        for name in args.workloads:
            w = wl.WORKLOADS[name]
            t0 = time.time()
            print(f"{name}: oracle on {args.jobs} processes", flush=True)
            if name.startswith("stream_"):
                write(name, stream_golden(w, pool))
            elif name.startswith("offline_"):
                for c in OFFLINE_CHUNKS_CHECKED:
                    write(f"{name}_chunk{c:02d}", batch_golden(wl.offline_chunk(w, c), pool, label=f"{name} chunk {c}"))
            else:
                write(name, batch_golden(w, pool))
            print(f"{name}: {time.time() - t0:.0f} s", flush=True)


if __name__ == "__main__":
    main()
