"""Benchmark of the kNN-LM mixture step on one MI355X.

A step is one knn_lm_mixture call (distances -> top-r -> softmax / scatter /
lambda-mix) over one batch of queries whose inputs already sit in HBM.  The
default workload is the Llama-2-7B-shaped decode query: B = 1, d = 4096,
N = 65536 bf16 keys (64 passages x 1024 tokens), r = 1024, V = 32000.  Two key
buffers of that shape alternate between steps so the 256 MB last-level cache
cannot serve a repeated key stream.

Prints one JSON line.  The dominant kernel (the distance stage) is timed with
HIP events around its launches inside the timed region, on the stream the
library launches on.  The CPU baseline is the fp64 oracle on a bounded sample
of the same workload on this host's cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0  # MI355X HBM3E, published
PEAK_MFMA_16BIT_TFLOPS = 2500.0  # MI355X dense bf16 / fp16 matrix cores, published
# The workloads of the per-config block, with the timed steps of each.
PER_CONFIG_STEPS = {"tiny": 200, "decode_7b": 200, "ragged_batch": 20, "decode_70b": 20, "specverify_seq": 10,
                    "specverify_static": 10}
# Workloads whose steps are also timed as replays of a HIP graph (steps short enough for the host's
# per-call launch work to show).
GRAPH_REPLAY = ("tiny", "decode_7b")
GRAPH_STEPS = 50  # steps captured in one graph
PMC_FILE = os.path.join(ROOT, "profiles", "dist_kernel_{workload}_pmc.json")
# The sources the distance kernels are built from (a change makes committed counters stale).
DIST_SOURCES = ("dist_kernels.hip", "mfma_kernels.hip", "mfma_packed.hip", "mfma_device.h", "knnlm_device.h",
                "knnlm_internal.h")


def _args():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", default="decode_7b")
    ap.add_argument("--packed-keys", action="store_true",
                    help="read the keys through their packed copy (knn_pack_keys; matrix-core workloads only)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of the oracle sample")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed region, run a plain 512 MiB device copy (HBM counter calibration)")
    ap.add_argument("--per-config", dest="per_config", action="store_true", default=None,
                    help="also time every workload (default: on for the decode_7b headline run)")
    ap.add_argument("--no-per-config", dest="per_config", action="store_false")
    return ap.parse_args()


def dist_kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in DIST_SOURCES:
        h.update(open(os.path.join(ROOT, "paper_2405_19325_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(workload):
    """HBM bytes per distance launch from committed rocprofv3 counters for this
    workload, if they were taken on this kernel source."""
    try:
        rec = json.load(open(PMC_FILE.format(workload=workload)))
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_hash") != dist_kernel_source_hash():
        return None
    return rec.get("hbm_bytes_per_launch")


def main():
    a = _args()
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {a.gpus} is not supported "
              "(the library's kNN-LM step has no cross-GPU path).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2405_19325_amd as knn
    from workloads import gen

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    spec = gen.config(a.workload)
    seed = gen.CONFIG_SEEDS[a.workload]
    w = gen.make(spec, seed, device=dev)
    keys2 = gen.second_key_copy(spec, seed, device=dev)
    hints = dict(key_offsets_host=w.key_offsets_host, query_offsets_host=w.query_offsets_host)
    packed = [knn.pack_keys(k) for k in (w.keys, keys2)] if a.packed_keys else [None, None]
    probs = [knn.MixtureProblem(w.queries, k, w.values, w.key_offsets, w.query_offsets, w.p_lm, w.r, w.mu, w.lam,
                                packed_keys=pk, **hints) for k, pk in zip((w.keys, keys2), packed)]
    torch.cuda.synchronize()

    B = spec.B
    total_keys = int(w.key_offsets_host[-1])
    esize = w.keys.element_size()
    # per-query key rows read: each query's own set (sets with several queries are read once)
    key_bytes = total_keys * spec.d * esize
    q_bytes = B * spec.d * esize
    dist_alg_bytes = key_bytes + q_bytes
    step_alg_bytes = dist_alg_bytes + 2 * B * spec.V * 4 + B * w.r * 4  # + p_LM in, p_M out, values gathered

    for i in range(a.warmup):
        probs[i % 2].run()
    torch.cuda.synchronize()

    # Every step is exactly what knn_lm_mixture enqueues (the distance stage, then
    # the fused select + mixture stage).  In every EVENT_EVERY-th step, HIP
    # events on the library's stream bracket the two launches to time the
    # dominant (distance) kernel live; an event record costs a few us, so the
    # other steps run without them.
    EVENT_EVERY = 8
    stream = torch.cuda.current_stream()
    n_ev = (a.steps + EVENT_EVERY - 1) // EVENT_EVERY
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n_ev)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for i in range(a.steps):
        p = probs[i % 2]
        if i % EVENT_EVERY == 0:
            e = ev[i // EVENT_EVERY]
            e[0].record(stream)
            p.run_part("distances")
            e[1].record(stream)
            p.run_part("select_mix")
            e[2].record(stream)
        else:
            p.run_part("distances")
            p.run_part("select_mix")
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    elapsed_ms = start.elapsed_time(end)
    dist_ms = [e[0].elapsed_time(e[1]) for e in ev]
    step_ms = [e[0].elapsed_time(e[2]) for e in ev]
    avg_dist_ms = sum(dist_ms) / len(dist_ms)
    avg_tail_ms = sum(s - d for s, d in zip(step_ms, dist_ms)) / len(step_ms)
    ms_per_step = elapsed_ms / a.steps
    qps = B * a.steps / (elapsed_ms / 1e3)

    # The distance stage alone, back to back on the same two key buffers, with
    # one pair of events around the whole run: its average launch time, free of
    # the few microseconds an event pair adds to a single launch.
    n_dist = min(a.steps, 200)
    d_start, d_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    d_start.record(stream)
    for i in range(n_dist):
        probs[i % 2].run_part("distances")
    d_end.record(stream)
    torch.cuda.synchronize()
    dist_launch_ms = d_start.elapsed_time(d_end) / n_dist

    # The distance and top-r stages alone (no mixture), the same way: the
    # path whose HBM efficiency the distance + select design is judged on.
    n_topr = min(a.steps, 200)
    t_start, t_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for i in range(4):
        probs[i % 2].run_part("distances")
        probs[i % 2].run_part("select")
    torch.cuda.synchronize()
    t_start.record(stream)
    for i in range(n_topr):
        probs[i % 2].run_part("distances")
        probs[i % 2].run_part("select")
    t_end.record(stream)
    torch.cuda.synchronize()
    topr_ms = t_start.elapsed_time(t_end) / n_topr
    topr = {"ms_per_step": round(topr_ms, 5), "alg_bytes": dist_alg_bytes + B * w.r * 8, "steps": n_topr,
            "hbm_frac": round((dist_alg_bytes + B * w.r * 8) / (topr_ms / 1e3) / 1e9 / PEAK_HBM_GBS, 4)}

    # The whole step with lambda_t per query from relative retrieval confidence
    # (alpha = 0.3, tau = 0.1) in place of the fixed lambda, the same way.
    n_rrc = min(a.steps, 200)
    r_start, r_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for i in range(4):
        probs[i % 2].run_rrc(0.3, 0.1)
    torch.cuda.synchronize()
    r_start.record(stream)
    for i in range(n_rrc):
        probs[i % 2].run_rrc(0.3, 0.1)
    r_end.record(stream)
    torch.cuda.synchronize()
    rrc_ms = r_start.elapsed_time(r_end) / n_rrc
    rrc = {"ms_per_step": round(rrc_ms, 5), "queries_per_s": round(B / (rrc_ms / 1e3), 1), "steps": n_rrc,
           "alpha": 0.3, "tau": 0.1}

    # One NEST decoding step (knn_nest_step: masked keys left out, lambda_t,
    # greedy token, span start, draft probability; then knn_spec_verify over
    # each set's rows as one draft), 1% of the keys masked, the p_LM argmax as
    # each row's draft token, the same way.
    n_nest = min(a.steps, 200)
    masked = np.random.default_rng(seed + 1).choice(total_keys, total_keys // 100, replace=False)
    mask = knn.mask_words(masked, total_keys, dev)
    draft = w.p_lm.argmax(1).to(torch.int32)
    offs = w.query_offsets
    for i in range(4):
        o = probs[i % 2].run_nest(0.3, 0.1, 0.5, key_mask=mask, draft_tokens=draft)
        knn.spec_verify(o["p_max"], o["p_draft"], o["next_token"], offs, 5e-2)
    torch.cuda.synchronize()
    n_start, n_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    n_start.record(stream)
    for i in range(n_nest):
        o = probs[i % 2].run_nest(0.3, 0.1, 0.5, key_mask=mask, draft_tokens=draft)
        knn.spec_verify(o["p_max"], o["p_draft"], o["next_token"], offs, 5e-2)
    n_end.record(stream)
    torch.cuda.synchronize()
    nest_ms = n_start.elapsed_time(n_end) / n_nest
    nest_step = {"ms_per_step": round(nest_ms, 5), "queries_per_s": round(B / (nest_ms / 1e3), 1), "steps": n_nest,
                 "alpha": 0.3, "tau": 0.1, "delta": 0.5, "gamma": 0.05, "masked_keys": int(len(masked))}

    # The key-norm pre-pass (knn_key_sqnorms, row (a1)): run once per datastore
    # before the decode loop, so it is reported apart from the step.
    # Algorithmic bytes: every key once, plus 4 bytes written per key.
    n_norm = min(a.steps, 50)
    norm_out = torch.empty(total_keys, dtype=torch.float32, device=dev)
    for i in range(2):
        knn.key_sqnorms(probs[i % 2].keys, out=norm_out)
    torch.cuda.synchronize()
    k_start, k_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    k_start.record(stream)
    for i in range(n_norm):
        knn.key_sqnorms(probs[i % 2].keys, out=norm_out)
    k_end.record(stream)
    torch.cuda.synchronize()
    norm_ms = k_start.elapsed_time(k_end) / n_norm
    norm_bytes = total_keys * (spec.d * w.keys.element_size() + 4)
    key_norms = {"ms_per_launch": round(norm_ms, 5), "alg_bytes": int(norm_bytes), "launches": n_norm,
                 "hbm_frac": round(norm_bytes / (norm_ms / 1e3) / 1e9 / PEAK_HBM_GBS, 4)}

    max_q = int(np.diff(w.query_offsets_host).max())
    matrix_core = spec.dtype in ("bf16", "f16") and spec.d % 8 == 0 and max_q >= 16
    achieved = dist_alg_bytes / (dist_launch_ms / 1e3) / 1e9
    traffic = measured_traffic(a.workload + ("_packed" if a.packed_keys else ""))
    kname = ("k_dist_packed" if a.packed_keys else "k_dist_mfma") if matrix_core else "k_dist_vec"
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": traffic,
                "kernel": "distance stage (" + kname + ")",
                "alg_bytes_per_launch": dist_alg_bytes,
                "avg_launch_ms": round(dist_launch_ms, 5), "timed_launches": n_dist,
                "in_step_event_ms": round(avg_dist_ms, 5)}

    stream_gbs = stream_read_gbs(knn, torch, dev)
    roofline["stream_read_gbs"] = round(stream_gbs, 1)
    roofline["frac_of_stream_read"] = round(achieved / stream_gbs, 4)

    if a.copy_calibration:
        src = torch.empty(256 * 1024 * 1024, dtype=torch.bfloat16, device=dev)  # 512 MiB
        src.fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()

    cpu = None
    if not a.no_cpu_baseline:
        cpu = cpu_baseline(w, spec, seed, a.cpu_seconds)

    per_config = None
    if a.per_config if a.per_config is not None else a.workload == "decode_7b":
        del probs, keys2, w
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        per_config = {name: time_config(name, steps, stream_gbs, not a.no_cpu_baseline)
                      for name, steps in PER_CONFIG_STEPS.items()}

    line = {
        "metric": "kNN-LM mixture queries/s + achieved HBM GB/s (d=4096, N=64K keys, r=1024)",
        "value": round(qps, 1),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec.dtype,
        "data": "synthetic (seeded N(0,1)*8/sqrt(d) keys and queries, Zipf(1.1) values, softmax N(0,2) p_LM)",
        "config": {
            "workload": (f"{spec.name}: B={B} queries, d={spec.d}, {spec.S} key set(s), N={total_keys} "
                         f"{spec.dtype} keys, r={spec.r}, V={spec.V}, mu={spec.mu:.6g}, lambda={spec.lam}"),
            "global_batch": B,
            "keys_per_query": total_keys // max(1, spec.S),
            "hidden": spec.d,
            "r": spec.r,
            "parallelism": "single GPU",
            "key_buffers_rotated": 2,
            "key_layout": "packed" if a.packed_keys else "row-major",
        },
        "select_mix_ms": round(avg_tail_ms, 5),
        "step_alg_bytes": step_alg_bytes,
        "step_hbm_frac": round(step_alg_bytes / (ms_per_step / 1e3) / 1e9 / PEAK_HBM_GBS, 4),
        "distance_topr": topr,
        "rrc_step": rrc,
        "nest_step": nest_step,
        "key_norms_prepass": key_norms,
        "host_wall_s": round(wall, 3),
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    if per_config is not None:
        line["per_config"] = per_config
    print(json.dumps(line), flush=True)


def stream_read_gbs(knn, torch, dev, nbytes=4 << 30, reps=10, trials=3):
    """HBM read rate of a plain read kernel (knn_stream_read) over a 4 GiB buffer, far larger than the last-level
    cache, the best of a few trials of back-to-back reads: the ceiling the distance stage's key streaming is
    compared with."""
    buf = torch.ones(nbytes // 2, dtype=torch.bfloat16, device=dev)
    sink = torch.zeros(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()
    for _ in range(3):
        knn.stream_read(buf, sink)
    best = float("inf")
    for _ in range(trials):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            knn.stream_read(buf, sink)
        e1.record(stream)
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1) / reps)
    del buf
    return nbytes / (best / 1e3) / 1e9


def _events_ms(torch, fn, n):
    """Average ms of fn(i) over n calls on the current stream (one event pair around all of them)."""
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for i in range(n):
        fn(i)
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / n


def _graph_ms(torch, fn, steps, replays):
    """Average ms per step of fn(0..steps-1) captured once in a HIP graph, over `replays` replays after an
    untimed one (the same work as the eager calls, without the host's per-call launches)."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        for i in range(steps):
            fn(i)
    torch.cuda.synchronize()
    graph.replay()
    ms = _events_ms(torch, lambda i: graph.replay(), replays) / steps
    del graph
    return ms


def time_config(name, steps, stream_gbs, with_oracle):
    """One workload at full size: the whole step, the distance stage alone and distance + top-r, each over
    `steps` back-to-back calls (two key buffers alternate when the keys would fit the last-level cache), the
    fractions of 8 TB/s (and of the measured plain read) on algorithmic bytes, the matrix cores' share of
    their dense peak on query batches, and the oracle's time for one query scaled by multiply-adds to the
    step."""
    import numpy as np
    import torch

    import paper_2405_19325_amd as knn
    from workloads import gen

    dev = torch.device("cuda:0")
    spec, seed = gen.config(name), gen.CONFIG_SEEDS[name]
    w = gen.make(spec, seed, device=dev)
    ko, qo = w.key_offsets_host, w.query_offsets_host
    nk, nq = np.diff(ko), np.diff(qo)
    esize = w.keys.element_size()
    total_keys = int(ko[-1])
    B = int(qo[-1])
    key_bytes = total_keys * spec.d * esize
    dist_bytes = key_bytes + B * spec.d * esize
    step_bytes = dist_bytes + 2 * B * spec.V * 4 + B * spec.r * 4
    topr_bytes = dist_bytes + B * spec.r * 8
    macs = int(np.sum(nq * nk)) * spec.d
    bufs = [w.keys]
    if key_bytes <= 4 * 256 * 2 ** 20:  # within a few times the 256 MB last-level cache
        bufs.append(gen.second_key_copy(spec, seed, device=dev))
    hints = dict(key_offsets_host=ko, query_offsets_host=qo)
    probs = [knn.MixtureProblem(w.queries, k, w.values, w.key_offsets, w.query_offsets, w.p_lm, w.r, w.mu, w.lam,
                                **hints) for k in bufs]
    nb = len(probs)
    for i in range(2):
        probs[i % nb].run()

    def full(i):
        probs[i % nb].run_part("distances")
        probs[i % nb].run_part("select_mix")

    def topr(i):
        probs[i % nb].run_part("distances")
        probs[i % nb].run_part("select")

    step_ms = _events_ms(torch, full, steps)
    dist_ms = _events_ms(torch, lambda i: probs[i % nb].run_part("distances"), steps)
    topr_ms = _events_ms(torch, topr, steps)
    dist_gbs = dist_bytes / (dist_ms / 1e3) / 1e9
    out = {
        "workload": (f"B={B}, d={spec.d}, {spec.S} key set(s), N={total_keys} {spec.dtype} keys, r={spec.r}, "
                     f"V={spec.V}"),
        "steps": steps,
        "ms_per_step": round(step_ms, 5),
        "queries_per_s": round(B / (step_ms / 1e3), 1),
        "step_alg_bytes": int(step_bytes),
        "step_hbm_frac": round(step_bytes / (step_ms / 1e3) / 1e9 / PEAK_HBM_GBS, 4),
        "distance_ms": round(dist_ms, 5),
        "distance_gbs": round(dist_gbs, 1),
        "distance_hbm_frac": round(dist_gbs / PEAK_HBM_GBS, 4),
        "distance_frac_of_stream_read": round(dist_gbs / stream_gbs, 4),
        "distance_topr_ms": round(topr_ms, 5),
        "distance_topr_hbm_frac": round(topr_bytes / (topr_ms / 1e3) / 1e9 / PEAK_HBM_GBS, 4),
        "key_buffers_rotated": nb,
    }
    if spec.dtype in ("bf16", "f16") and spec.d % 128 == 0 and int(nq.max()) >= 16:
        tflops = 2.0 * macs / (dist_ms / 1e3) / 1e12
        out["matrix_cores"] = {"alg_flops": 2 * macs, "tflops": round(tflops, 1),
                               "frac_of_dense_peak": round(tflops / PEAK_MFMA_16BIT_TFLOPS, 4)}
        out["packed_keys"] = time_packed(knn, torch, w, bufs, hints, steps, dist_bytes, step_bytes)
    if name in GRAPH_REPLAY:
        g_ms = _graph_ms(torch, full, GRAPH_STEPS, max(steps // GRAPH_STEPS, 2))
        out["graph_replay"] = {"steps_per_graph": GRAPH_STEPS, "ms_per_step": round(g_ms, 5),
                               "queries_per_s": round(B / (g_ms / 1e3), 1),
                               "step_hbm_frac": round(step_bytes / (g_ms / 1e3) / 1e9 / PEAK_HBM_GBS, 4)}
    del probs, bufs
    if with_oracle:
        out["oracle"] = oracle_estimate(w, spec, macs)
    del w
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def time_packed(knn, torch, w, bufs, hints, steps, dist_bytes, step_bytes):
    """The same workload over the packed copy of its keys (knn_pack_keys, run once per key store and timed
    apart): the distance stage and the whole step, as above."""
    packed = [knn.pack_keys(k) for k in bufs]
    pack_ms = _events_ms(torch, lambda i: knn.pack_keys(bufs[0], out=packed[0]), 2)
    probs = [knn.MixtureProblem(w.queries, k, w.values, w.key_offsets, w.query_offsets, w.p_lm, w.r, w.mu, w.lam,
                                packed_keys=pk, **hints) for k, pk in zip(bufs, packed)]
    nb = len(probs)
    for i in range(2):
        probs[i % nb].run()

    def full(i):
        probs[i % nb].run_part("distances")
        probs[i % nb].run_part("select_mix")

    step_ms = _events_ms(torch, full, steps)
    dist_ms = _events_ms(torch, lambda i: probs[i % nb].run_part("distances"), steps)
    out = {"pack_ms": round(pack_ms, 3), "packed_bytes": int(packed[0].numel()),
           "ms_per_step": round(step_ms, 5), "queries_per_s": round(w.spec.B / (step_ms / 1e3), 1),
           "step_hbm_frac": round(step_bytes / (step_ms / 1e3) / 1e9 / PEAK_HBM_GBS, 4),
           "distance_ms": round(dist_ms, 5),
           "distance_hbm_frac": round(dist_bytes / (dist_ms / 1e3) / 1e9 / PEAK_HBM_GBS, 4)}
    del probs, packed
    return out


def oracle_estimate(w, spec, step_macs):
    """The fp64 oracle (select + mix) on the workload's first query against its own key set, timed on this
    host, and that time scaled by multiply-adds to the whole step."""
    import numpy as np

    import oracle

    threads = host_threads()
    ko, qo = w.key_offsets_host, w.query_offsets_host
    s = int(np.searchsorted(qo, 0, side="right") - 1)
    n = int(ko[s + 1] - ko[s])
    keys_h, dt = oracle.host_elements(w.keys[ko[s]:ko[s + 1]])
    q_h, _ = oracle.host_elements(w.queries[:1])
    vals = w.values[ko[s]:ko[s + 1]].cpu().numpy()
    p_lm = w.p_lm[:1].cpu().numpy()
    k1, q1 = np.array([0, n], dtype=np.int64), np.array([0, 1], dtype=np.int64)
    t0 = time.perf_counter()
    ids, dists = oracle.select(q_h, keys_h, dt, k1, q1, spec.r, nthreads=threads)
    oracle.mix(ids, dists, vals, k1, q1, p_lm, spec.mu, spec.lam)
    el = time.perf_counter() - t0
    q_macs = n * spec.d
    return {"one_query_s": round(el, 3), "one_query_macs": int(q_macs),
            "est_s_per_step": round(el * step_macs / q_macs, 2), "cores": threads}


def host_threads():
    """Threads the oracle uses: every core this process may run on, at most 16 (one GPU's share of the host)."""
    return max(1, min(16, len(os.sched_getaffinity(0))))


def cpu_baseline(w, spec, seed, budget_s):
    """The fp64 oracle on a bounded sample: further decode queries against the same key set."""
    import numpy as np

    import oracle
    from workloads import gen

    threads = host_threads()
    n0 = int(w.key_offsets_host[1])  # the sample queries the first key set
    keys_h, dt = oracle.host_elements(w.keys[:n0])
    vals = w.values[:n0].cpu().numpy()
    ko, qo1 = np.array([0, n0], dtype=np.int64), np.array([0, 1], dtype=np.int64)
    extra = gen.extra_queries(spec, seed, 4096, device="cpu")
    q_all, _ = oracle.host_elements(extra)
    p_lm = w.p_lm[:1].cpu().numpy()
    done = 0
    t0 = time.perf_counter()
    while done < q_all.shape[0]:
        q1 = q_all[done:done + 1]
        ids, dists = oracle.select(q1, keys_h, dt, ko, qo1, spec.r, nthreads=threads)
        oracle.mix(ids, dists, vals, ko, qo1, p_lm, spec.mu, spec.lam)
        done += 1
        if time.perf_counter() - t0 > budget_s:
            break
    el = time.perf_counter() - t0
    return {"value": round(done / el, 3), "unit": "queries/s", "cores": threads, "kind": "oracle",
            "nproc": len(os.sched_getaffinity(0)), "cpu_model": _cpu_model(),
            "sample": (f"{done} decode queries of the same shape (d={spec.d}, one set of {n0} keys, "
                       f"r={spec.r}) through the fp64 oracle select + mix, {el:.1f} s wall, {threads} threads "
                       f"(every core this process may use, at most 16); CPU: {_cpu_model()}")}


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


if __name__ == "__main__":
    main()
