#!/usr/bin/env python3
"""Throughput of the A-PACK prune path on one MI355X.

Workload: a 5-minute clip at the Qwen2.5-Omni-7B shape (7500 audio + 600x144
visual + 128 text tokens; 28 query / 4 KV heads, head dim 128, hidden 3584,
bf16) with a 28-layer K/V cache.  One step prunes at layers 14, 18 and 22
with cumulative keep 0.7, 0.5 and 0.3 of the original audio and visual
counts; each prune (GQA scores over the candidates, per-modality top-k,
kept-row list) is followed by the compaction of all 28 layers' K/V, the
hidden states and the position ids.  Inputs are synthetic and resident in
HBM before timing starts.

Prints one JSON line: candidate tokens entering a prune step per second
(whole job), with the HBM roofline of the dominant kernel (the gather
compaction, timed with HIP events on the launch stream) and the fp64 CPU
oracle timed on a bounded sample on this host.
"""

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "pruned tokens/sec (score+top-k+KV compact) at 7B shape; achieved HBM GB/s"
HBM_PEAK_GBS = 8000.0


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def measured_traffic():
    """Per-launch HBM bytes of k_gather from the committed rocprofv3 counter
    summary, or None when the gather source has changed since it was taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "k_gather_traffic_progressive7b.md")
    try:
        text = open(path).read()
    except OSError:
        return None
    vals = {}
    for line in text.splitlines():
        line = line.strip()
        for key in ("traffic_bytes_per_launch", "source", "source_sha256"):
            if line.startswith(key + ":"):
                vals[key] = line.split(":", 1)[1].strip()
    try:
        src = open(os.path.join(ROOT, vals["source"]), "rb").read()
    except (KeyError, OSError):
        return None
    if hashlib.sha256(src).hexdigest() != vals.get("source_sha256"):
        return None
    return float(vals["traffic_bytes_per_launch"])


def to_dev(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).cuda()


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the CPU oracle timing")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB mebibytes three times (reference for HBM "
                         "byte counters) and exit")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the prune path needs no collective, and runs with "
              "--gpus > 1 are not part of this build", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_08794_amd as A
    import workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    A.library()
    torch.cuda.set_device(0)
    if args.copy_calibration:
        n = args.copy_calibration * (1 << 20)
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "copies": 3}))
        return

    t0 = time.time()
    case = W.progressive_case()
    log(f"generated workload in {time.time() - t0:.1f}s")
    cache = case.cache
    n_layers = len(cache.k_layers)
    seq = case.seq()
    n0 = seq.n_tokens
    hkv, d, hid = case.hkv, case.d, case.hidden_dim

    # Device buffers: the full cache plus one output cache per prune step.
    k_in = [to_dev(x) for x in cache.k_layers]
    v_in = [to_dev(x) for x in cache.v_layers]
    h_in = to_dev(cache.hidden)
    p_in = torch.from_numpy(cache.pos).cuda()
    queries = [to_dev(x) for x in case.queries]
    # Step descriptors: the cumulative keep counts against the original counts.
    steps = []
    n_cur = n0
    spans_cur = list(seq.spans)
    n_a, n_v = case.n_audio, case.n_visual
    for layer, keep in zip(case.prune_layers, case.keeps):
        s = W.PruneSeq(0, n_cur, spans_cur, 0, case.q_len, (keep, keep), (n_a, n_v))
        n_kept, ws_bytes = A.apack_prune_layer_query([s], case.hq, hkv, d)
        n_out = n_kept[0]
        ka = A.apack_keep_count(keep, n_a)
        kv = A.apack_keep_count(keep, n_v)
        steps.append(dict(layer=layer, seq=s, n_in=n_cur, n_out=n_out, cand=n_cur - case.n_text,
                          ws=torch.empty(ws_bytes, dtype=torch.uint8, device="cuda"),
                          scores=torch.empty(n_cur, dtype=torch.float32, device="cuda"),
                          kept=torch.empty(n_out, dtype=torch.int32, device="cuda"),
                          k_out=[torch.empty((hkv, n_out, d), dtype=torch.bfloat16, device="cuda")
                                 for _ in range(n_layers)],
                          v_out=[torch.empty((hkv, n_out, d), dtype=torch.bfloat16, device="cuda")
                                 for _ in range(n_layers)],
                          h_out=torch.empty((n_out, hid), dtype=torch.bfloat16, device="cuda"),
                          p_out=torch.empty((3, n_out), dtype=torch.int32, device="cuda")))
        spans_cur = [(0, ka, W.AUDIO), (ka, kv, W.VISUAL)]
        n_cur = n_out
    torch.cuda.synchronize()
    log(f"uploaded {sum(x.numel() * 2 for x in k_in + v_in) / 1e9:.2f} GB cache in {time.time() - t0:.1f}s")

    def events():
        return [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in steps]

    def run_step(ev):
        kk, vv, hh, pp = k_in, v_in, h_in, p_in
        for i, st in enumerate(steps):
            if ev:
                ev[i][0].record()
            A.apack_prune_layer(queries[i], kk[st["layer"]], [st["seq"]], scores=st["scores"],
                                kept_rows=st["kept"], workspace=st["ws"])
            if ev:
                ev[i][1].record()
                ev[i][2].record()
            A.apack_compact_kv(st["kept"], st["n_in"], kk, vv, st["k_out"], st["v_out"], hh, st["h_out"],
                               pp, st["p_out"])
            if ev:
                ev[i][3].record()
            kk, vv, hh, pp = st["k_out"], st["v_out"], st["h_out"], st["p_out"]

    for _ in range(args.warmup):
        run_step(None)
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")

    # Every timed step records its own events on the launch stream; they are
    # read only after the timed region.
    step_events = [events() for _ in range(args.steps)]
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for ev in step_events:
        run_step(ev)
    stop.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(stop)
    ms_per_step = total_ms / args.steps
    prune_ms = [sum(ev[i][0].elapsed_time(ev[i][1]) for ev in step_events) for i in range(len(steps))]
    gather_ms = [sum(ev[i][2].elapsed_time(ev[i][3]) for ev in step_events) for i in range(len(steps))]
    log(f"timed {args.steps} steps: {ms_per_step:.3f} ms/step")

    # Throughput and algorithmic bytes.
    cand_per_step = sum(st["cand"] for st in steps)
    removed = sum(st["n_in"] - st["n_out"] for st in steps)
    e = 2
    row_bytes = n_layers * 2 * hkv * d * e + hid * e + 3 * 4   # K/V of every layer, hidden, 3 position ids
    gather_bytes = [st["n_out"] * (2 * row_bytes + 4) for st in steps]
    score_bytes = [st["cand"] * hkv * d * e + case.hq * case.q_len * d * e + 4 * st["n_in"] + 4 * st["n_out"]
                   for st in steps]
    step_bytes = sum(gather_bytes) + sum(score_bytes)
    value = cand_per_step / (ms_per_step / 1e3)
    g_ms = [x / args.steps for x in gather_ms]
    p_ms = [x / args.steps for x in prune_ms]
    achieved = sum(gather_bytes) / (sum(g_ms) / 1e3) / 1e9
    result = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "candidate tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "progressive prune of a 5-min clip, 7B shape: 7500 audio + 600x144 visual + 128 text "
                        "tokens, 28/4 heads, head dim 128, hidden 3584, 28-layer cache, prune layers 14/18/22 "
                        "at cumulative keep 0.7/0.5/0.3",
            "tokens": n0, "candidates_per_step": cand_per_step, "removed_per_step": removed,
            "layers": n_layers, "query_rows": case.q_len,
        },
        "achieved_hbm_gbs": round(step_bytes / (ms_per_step / 1e3) / 1e9, 1),
        "removed_tokens_per_s": round(removed / (ms_per_step / 1e3), 1),
        "roofline": {
            "bound": "hbm",
            "kernel": "k_gather",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic(),
            "algorithmic_bytes_per_launch": round(sum(gather_bytes) / len(gather_bytes)),
        },
        "per_prune_step_ms": {"score_select": [round(x, 4) for x in p_ms], "compact": [round(x, 4) for x in g_ms]},
        "algorithmic_bytes_per_step": step_bytes,
    }

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(case, steps[0])
    print(json.dumps(result), flush=True)


def cpu_baseline(case, st):
    """fp64 oracle on prune step 1 of the same workload (bounded sample)."""
    from threadpoolctl import threadpool_info
    from oracle import prune as OP, widen

    s = st["seq"]
    t0 = time.perf_counter()
    q = widen(case.queries[0], "bf16")
    k = widen(case.cache.k_layers[st["layer"]], "bf16")
    r = OP.prune_sequence(q, k, s.tags(), s.keep, s.keep_basis)
    kept = r["kept"]
    for x in case.cache.k_layers + case.cache.v_layers:
        OP.compact_rows(x, kept, axis=1)
    OP.compact_rows(case.cache.hidden, kept, axis=0)
    OP.compact_rows(case.cache.pos, kept, axis=1)
    dt = time.perf_counter() - t0
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    log(f"cpu oracle step 1: {dt:.1f}s")
    return {
        "value": round(st["cand"] / dt, 1),
        "unit": "candidate tokens/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"prune step 1 of 3 ({st['cand']} candidates): fp64 scores, top-k and the gather of all "
                  f"28 layers' K/V, hidden states and positions; {dt:.1f} s on {os.cpu_count()} host CPUs",
    }


if __name__ == "__main__":
    main()
