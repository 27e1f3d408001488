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
    ap.add_argument("--no-other-configs", action="store_true", help="skip the config 2 and 3 measurements")
    ap.add_argument("--no-ragged", action="store_true", help="skip the ragged batch of 8 clips (config 5)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB mebibytes three times (reference for HBM "
                         "byte counters) and exit")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the prune path needs no collective, and runs on "
              "more than one GPU (--gpus > 1) are not implemented", file=sys.stderr)
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

    # Per prune step two events: after its scores/select (= before its gather)
    # and after its gather (= before the next prune).  Neighbouring phases share
    # an event, so a step records 6 markers rather than 12.
    def events():
        return [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in steps]

    def run_step(ev):
        kk, vv, hh, pp = k_in, v_in, h_in, p_in
        for i, st in enumerate(steps):
            A.apack_prune_layer(queries[i], kk[st["layer"]], [st["seq"]], scores=st["scores"],
                                kept_rows=st["kept"], workspace=st["ws"])
            if ev:
                ev[i][0].record()
            A.apack_compact_kv(st["kept"], st["n_in"], kk, vv, st["k_out"], st["v_out"], hh, st["h_out"],
                               pp, st["p_out"])
            if ev:
                ev[i][1].record()
            kk, vv, hh, pp = st["k_out"], st["v_out"], st["h_out"], st["p_out"]

    for _ in range(args.warmup):
        run_step(None)
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")

    # The timed steps carry no markers between their launches (on some runs
    # each timing event between two kernels cost ~9 us); the phases are timed
    # in a second pass of the same K steps, each step recording its own events
    # on the launch stream, read only after that pass.
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        run_step(None)
    stop.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(stop)
    ms_per_step = total_ms / args.steps
    log(f"timed {args.steps} steps: {ms_per_step:.3f} ms/step")
    step_events = [events() for _ in range(args.steps)]
    start_p = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start_p.record()
    for ev in step_events:
        run_step(ev)
    torch.cuda.synchronize()
    # The scores/select phase of prune i runs from the previous gather's end
    # (the step's start for the first prune) to the event after it.
    prev = [start_p] + [ev[-1][1] for ev in step_events[:-1]]
    prune_ms = [sum((p if i == 0 else ev[i - 1][1]).elapsed_time(ev[i][0]) for p, ev in zip(prev, step_events))
                for i in range(len(steps))]
    gather_ms = [sum(ev[i][0].elapsed_time(ev[i][1]) for ev in step_events) for i in range(len(steps))]
    phase_ms = start_p.elapsed_time(step_events[-1][-1][1]) / args.steps
    log(f"phase pass: {phase_ms:.3f} ms/step with its markers")
    cold_ms = cold_steps(torch, run_step, args.steps)
    log(f"cold: {cold_ms:.3f} ms/step")

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
        "headline_cold": {
            "ms_per_step": round(cold_ms, 4),
            "value": round(cand_per_step / (cold_ms / 1e3), 1),
            "achieved_hbm_gbs": round(step_bytes / (cold_ms / 1e3) / 1e9, 1),
            "how": "the same K steps, each after a 512 MiB device write (twice the Infinity Cache) that lies "
                   "outside its events; value and ms_per_step above are the back-to-back (warm) steps",
        },
        "per_prune_step_ms": {"score_select": [round(x, 4) for x in p_ms], "compact": [round(x, 4) for x in g_ms],
                              "how": "a second pass of the same steps with an event after each select and each "
                                     "gather; that pass took %.4f ms per step" % phase_ms},
        "prefill_flops": prefill_flops(A, n_layers, n0, case.prune_layers, [st["n_out"] for st in steps]),
        "algorithmic_bytes_per_step": step_bytes,
    }

    if not args.no_other_configs:
        result["in_place_compaction"] = in_place_compaction(torch, A, steps, k_in, v_in, h_in, p_in, row_bytes,
                                                            g_ms)
        del k_in, v_in, h_in, p_in, queries, steps
        torch.cuda.empty_cache()
        result["other_configs"] = other_configs(torch, A, W, not args.no_ragged)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(case)
    print(json.dumps(result), flush=True)


def cold_steps(torch, run_step, steps):
    """Mean device time of `steps` steps, each started after a 512 MiB write
    that evicts the Infinity Cache; the write lies outside the step's
    events."""
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    total = 0.0
    for _ in range(steps):
        flush.fill_(1)
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        run_step(None)
        b.record()
        torch.cuda.synchronize()
        total += a.elapsed_time(b)
    del flush
    return total / steps


def _time_calls(torch, fn, flush, reps=20, warmup=5):
    """Median device time of fn() over reps, cold (a 512 MiB write before
    each repetition evicts the 256 MB Infinity Cache) and warm."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    out = {}
    for mode in ("cold", "warm"):
        ms = []
        for _ in range(reps):
            if mode == "cold":
                flush.fill_(1)
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            ms.append(a.elapsed_time(b))
        out[mode] = float(np.median(ms))
    return out


def prefill_flops(A, n_layers, n0, prune_layers, n_after, d_model=3584, d_ffn=18944):
    """Analytic prefill FLOPs (Appendix G) of the schedule the run produced:
    each prune takes effect from the layer after it, at the kept counts the
    prune calls returned; 7B thinker constants."""
    lengths = A.apack_schedule_lengths(n_layers, n0, prune_layers, n_after)
    f_pre, ratio = A.apack_prefill_flops(lengths, n0, d_model, d_ffn)
    return {"f_pre_tflops": round(f_pre / 1e12, 3),
            "full_tflops": round(n_layers * A.apack_layer_flops(n0, d_model, d_ffn) / 1e12, 3),
            "ratio": round(ratio, 4), "final_retention": round(lengths[-1] / n0, 4)}


def in_place_compaction(torch, A, steps, k_in, v_in, h_in, p_in, row_bytes, gather_ms):
    """The step's three compactions done in place on one cache with the kept
    lists of the timed run: per launch, the median time (cold and warm, 10
    repetitions after 2 warm-ups) against the out-of-place gather.  Repeating
    a compaction in place shuffles the cache's contents but not the work.
    Rows whose index does not change (the kept prefix) are not moved, so the
    algorithmic bytes count only the rows that move."""
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    ws = torch.empty(A.apack_compact_kv_inplace_workspace(steps[0]["n_out"]), dtype=torch.uint8, device="cuda")
    out = []
    for i, st in enumerate(steps):
        n = st["n_in"]
        view = ([x[:, :n] for x in k_in], [x[:, :n] for x in v_in], h_in[:n], p_in[:, :n])
        kept = st["kept"].cpu().numpy()
        moved = int(np.count_nonzero(kept != np.arange(kept.size)))
        nbytes = moved * 2 * row_bytes + 4 * kept.size
        t = _time_calls(torch, lambda: A.apack_compact_kv_inplace(st["kept"], n, *view, workspace=ws), flush,
                        reps=10, warmup=2)
        out.append({"rows_in": n, "rows_out": int(kept.size), "rows_moved": moved, "algorithmic_bytes": nbytes,
                    "ms_cold": round(t["cold"], 4), "ms_warm": round(t["warm"], 4),
                    "achieved_gbs_cold": round(nbytes / (t["cold"] / 1e3) / 1e9, 1),
                    "out_of_place_gather_ms": round(gather_ms[i], 4)})
    log("in-place compaction: " + ", ".join(f"{o['ms_cold']:.3f} ms ({o['achieved_gbs_cold']:.0f} GB/s)"
                                            for o in out))
    return out


def _prune_bytes(case, n_kept, n_layers, hidden_dim, e=2):
    """Algorithmic bytes of one prune + compaction: K over S, Q, scores and
    kept rows written, one read and one write of every kept row's K/V,
    hidden state and position ids, and one read of the kept list."""
    cand = sum(int((s.tags() != 0).sum()) for s in case.seqs)
    q_rows = sum(s.q_len for s in case.seqs)
    row = n_layers * 2 * case.hkv * case.d * e + hidden_dim * e + 3 * 4
    return cand, (cand * case.hkv * case.d * e + case.hq * q_rows * case.d * e + 4 * cand + 4 * n_kept
                  + n_kept * (2 * row + 4))


def other_configs(torch, A, W, with_ragged):
    """Configs 2, 3 and 5 (unless --no-ragged): the whole launch sequence timed
    as one, median of 20 after 5 warm-ups, cold and warm."""
    import workloads as W  # noqa: F811
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    res = {}

    def dev(x):
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).cuda()

    def prune_compact(case, cache):
        q, k = dev(case.q), dev(case.k)
        v, hid = dev(cache.v_layers[0]), dev(cache.hidden)
        pos = torch.from_numpy(cache.pos).cuda()
        n_kept, wsb = A.apack_prune_layer_query(case.seqs, case.hq, case.hkv, case.d)
        n_out = int(sum(n_kept))
        ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
        sc = torch.empty(k.shape[1], dtype=torch.float32, device="cuda")
        kept = torch.empty(n_out, dtype=torch.int32, device="cuda")
        k_out = torch.empty((case.hkv, n_out, case.d), dtype=k.dtype, device="cuda")
        v_out = torch.empty_like(k_out)
        h_out = torch.empty((n_out, hid.shape[1]), dtype=hid.dtype, device="cuda")
        p_out = torch.empty((3, n_out), dtype=torch.int32, device="cuda")

        def run():
            A.apack_prune_layer(q, k, case.seqs, scores=sc, kept_rows=kept, workspace=ws)
            A.apack_compact_kv(kept, k.shape[1], [k], [v], [k_out], [v_out], hid, h_out, pos, p_out)
        return run, n_out, hid.shape[1]

    def scorer(dyn):
        xv, xa, xq = dev(dyn.xv), dev(dyn.xa), dev(dyn.xq)
        n_kv, wsb = A.apack_score_dynamics_query(dyn.seqs, dyn.dim, dyn.params)
        ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
        nk = int(sum(n_kv))
        emb = torch.empty((nk, xv.shape[1]), dtype=xv.dtype, device="cuda")
        bytes_ = 2 * (xv.numel() + xa.numel() + xq.numel()) + 2 * 2 * nk * xv.shape[1]

        def run():
            out = A.apack_score_dynamics(xv, xa, xq, dyn.seqs, dyn.params, workspace=ws)
            A.apack_compact_kv(out["kept"], xv.shape[0], hidden_in=xv, hidden_out=emb)
        return run, bytes_

    def entry(t, cand, nbytes, what):
        return {"what": what, "candidates": cand, "algorithmic_bytes": int(nbytes),
                "ms_cold": round(t["cold"], 4), "ms_warm": round(t["warm"], 4),
                "candidate_tokens_per_s_cold": round(cand / (t["cold"] / 1e3), 1),
                "achieved_gbs_cold": round(nbytes / (t["cold"] / 1e3) / 1e9, 1)}

    t0 = time.time()
    case = W.prune_cfg2()
    cache = W.cfg_cache(2, case)
    run, n_out, hd = prune_compact(case, cache)
    cand, nb = _prune_bytes(case, n_out, 1, hd)
    res["cfg2_3b_layer"] = entry(_time_calls(torch, run, flush), cand, nb,
                                 "prune + compaction of one layer's K/V, hidden states and positions")
    log(f"config 2 done ({time.time() - t0:.1f}s)")

    dyn = W.dynamics_cfg3("offset")
    case = W.prune_cfg3()
    cache = W.cfg_cache(3, case)
    s_run, s_bytes = scorer(dyn)
    p_run, n_out, hd = prune_compact(case, cache)
    cand, nb = _prune_bytes(case, n_out, 1, hd)
    ts = _time_calls(torch, s_run, flush)
    tp = _time_calls(torch, p_run, flush)
    res["cfg3_7b_scorer_gate_on"] = entry(ts, int(dyn.xv.shape[0]), s_bytes,
                                          "pre-LLM scorer of a 60 s clip (gate fired) + gather of the kept "
                                          "visual embeddings")
    res["cfg3_7b_prune"] = entry(tp, cand, nb, "in-LLM prune + one-layer compaction of the 9454-row sequence")
    res["cfg3_7b_scorer_alignments"] = alignment_ablation(torch, A, dyn, flush, dev)
    log(f"config 3 done ({time.time() - t0:.1f}s)")

    res["paper_schedule_7b"] = paper_schedule(torch, A, W, flush, dev)
    log(f"paper schedule done ({time.time() - t0:.1f}s)")

    if with_ragged:
        rb = W.ragged_batch()
        log(f"ragged batch generated ({time.time() - t0:.1f}s)")
        s_run, s_bytes = scorer(rb.dynamics)
        p_run, n_out, hd = prune_compact(rb.prune, rb.cache)
        cand, nb = _prune_bytes(rb.prune, n_out, 1, hd)

        def both():
            s_run()
            p_run()
        t = _time_calls(torch, both, flush)
        res["cfg5_ragged_8_clips"] = entry(t, cand, nb + s_bytes,
                                           f"scorer + embedding gather + prune + compaction of 8 clips of "
                                           f"{rb.seconds} s, one launch sequence")
        log(f"config 5 done ({time.time() - t0:.1f}s)")
    return res


def alignment_ablation(torch, A, dyn, flush, dev):
    """The alternative frame-alignment scorers on the 60 s 7B clip whose
    window CKA is low (the gate fires): scorer time, and how many kept
    visual tokens each shares with the paper's gated CKA."""
    xv, xa, xq = dev(dyn.xv), dev(dyn.xa), dev(dyn.xq)
    kept, out = {}, {}
    for name in ("gated_cka", "cka", "av_cosine", "spatial_cka"):
        params = dict(dyn.params, alignment=name)
        n_kv, wsb = A.apack_score_dynamics_query(dyn.seqs, dyn.dim, params)
        ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
        t = _time_calls(torch, lambda: A.apack_score_dynamics(xv, xa, xq, dyn.seqs, params, workspace=ws), flush,
                        reps=10, warmup=2)
        r = A.apack_score_dynamics(xv, xa, xq, dyn.seqs, params, workspace=ws)
        torch.cuda.synchronize()
        kept[name] = set(r["kept"].cpu().numpy().tolist())
        out[name] = {"ms_cold": round(t["cold"], 4), "gate_fired": bool(r["gate"].cpu().numpy()[0]),
                     "kept": len(kept[name])}
    for name in out:
        out[name]["kept_shared_with_gated_cka"] = round(len(kept[name] & kept["gated_cka"]) / max(1, len(kept[name])),
                                                        4)
    return out


def paper_schedule(torch, A, W, flush, dev):
    """Eq. 6 as the paper writes it, on the 5-minute 7B clip: from layer 14
    on, every layer keeps the top ceil(0.9 |S|) of the current candidates,
    ranked jointly by the last query token, and compacts all 28 layers' K/V,
    the hidden states and the positions.  Joint ranking ignores modality, so
    each step's candidates are one span; no host synchronisation between
    steps."""
    pc = W.paper_schedule_case()
    hkv, d, hid = pc.hkv, pc.d, pc.hidden_dim
    n_layers = len(pc.cache.k_layers)
    k_in = [dev(x) for x in pc.cache.k_layers]
    v_in = [dev(x) for x in pc.cache.v_layers]
    h_in = dev(pc.cache.hidden)
    p_in = torch.from_numpy(pc.cache.pos).cuda()
    qs = [dev(x) for x in pc.queries]
    n_text = pc.n_text
    steps, n_cand = [], pc.n_audio + pc.n_visual
    for keep in pc.keeps:
        seq = W.PruneSeq(0, n_cand + n_text, [(0, n_cand, W.AUDIO)], 0, 1, (keep, 0.0), (0, 0), True)
        n_kept, wsb = A.apack_prune_layer_query([seq], pc.hq, hkv, d)
        steps.append(dict(seq=seq, n_in=n_cand + n_text, n_out=n_kept[0], cand=n_cand,
                          ws=torch.empty(wsb, dtype=torch.uint8, device="cuda"),
                          scores=torch.empty(n_cand + n_text, dtype=torch.float32, device="cuda"),
                          kept=torch.empty(n_kept[0], dtype=torch.int32, device="cuda")))
        n_cand = n_kept[0] - n_text
    m = steps[0]["n_out"]
    bufs = [dict(k=[torch.empty((hkv, m, d), dtype=torch.bfloat16, device="cuda") for _ in range(n_layers)],
                 v=[torch.empty((hkv, m, d), dtype=torch.bfloat16, device="cuda") for _ in range(n_layers)],
                 h=torch.empty((m, hid), dtype=torch.bfloat16, device="cuda"),
                 p=torch.empty((3, m), dtype=torch.int32, device="cuda")) for _ in range(2)]

    def run():
        kk, vv, hh, pp = k_in, v_in, h_in, p_in
        for i, (layer, st) in enumerate(zip(pc.prune_layers, steps)):
            A.apack_prune_layer(qs[i], kk[layer], [st["seq"]], scores=st["scores"], kept_rows=st["kept"],
                                workspace=st["ws"])
            b, r = bufs[i % 2], st["n_out"]
            ko = [x[:, :r] for x in b["k"]]
            vo = [x[:, :r] for x in b["v"]]
            A.apack_compact_kv(st["kept"], st["n_in"], kk, vv, ko, vo, hh, b["h"][:r], pp, b["p"][:, :r])
            kk, vv, hh, pp = ko, vo, b["h"][:r], b["p"][:, :r]
    t = _time_calls(torch, run, flush, reps=10, warmup=3)
    e = 2
    row = n_layers * 2 * hkv * d * e + hid * e + 3 * 4
    cand = sum(st["cand"] for st in steps)
    nbytes = sum(st["cand"] * hkv * d * e + pc.hq * d * e + 4 * st["n_in"] + 4 * st["n_out"]
                 + st["n_out"] * (2 * row + 4) for st in steps)
    return {"what": f"paper schedule: joint top-k, last query only, drop 10% at each of layers "
                    f"{pc.prune_layers[0]}-{pc.prune_layers[-1]} of a 5-min 7B clip, each step compacting all "
                    f"{n_layers} layers",
            "candidates": cand, "algorithmic_bytes": int(nbytes),
            "ms_cold": round(t["cold"], 3), "ms_warm": round(t["warm"], 3),
            "candidate_tokens_per_s_cold": round(cand / (t["cold"] / 1e3), 1),
            "achieved_gbs_cold": round(nbytes / (t["cold"] / 1e3) / 1e9, 1),
            "prefill_flops": prefill_flops(A, n_layers, pc.seq().n_tokens, list(pc.prune_layers),
                                           [st["n_out"] for st in steps])}


def cpu_baseline(case, repeats=3):
    """The fp64 oracle on one whole step of the same workload (three prune
    steps, each with the gather of all 28 layers' K/V, the hidden states and
    the positions), best of `repeats` runs."""
    from threadpoolctl import threadpool_info
    import workloads as W
    from oracle import prune as OP, widen

    times = []
    cand = 0
    for _ in range(repeats):
        t0 = time.perf_counter()
        cand = 0
        k_layers, v_layers, hidden, pos = case.cache.k_layers, case.cache.v_layers, case.cache.hidden, case.cache.pos
        seq = case.seq()
        n_a, n_v = case.n_audio, case.n_visual
        spans, n = list(seq.spans), seq.n_tokens
        for i, (layer, keep) in enumerate(zip(case.prune_layers, case.keeps)):
            s = W.PruneSeq(0, n, spans, 0, case.q_len, (keep, keep), (n_a, n_v))
            q = widen(case.queries[i], "bf16")
            k = widen(k_layers[layer], "bf16")
            r = OP.prune_sequence(q, k, s.tags(), s.keep, s.keep_basis)
            kept = r["kept"]
            cand += int((s.tags() != 0).sum())
            k_layers = [OP.compact_rows(x, kept, axis=1) for x in k_layers]
            v_layers = [OP.compact_rows(x, kept, axis=1) for x in v_layers]
            hidden = OP.compact_rows(hidden, kept, axis=0)
            pos = OP.compact_rows(pos, kept, axis=1)
            ka, kv = r["k"]["audio"], r["k"]["visual"]
            spans, n = [(0, ka, W.AUDIO), (ka, kv, W.VISUAL)], len(kept)
        times.append(time.perf_counter() - t0)
    dt = min(times)
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    log(f"cpu oracle: {', '.join(f'{t:.1f}' for t in times)} s per step")
    single = single_thread_configs(OP, widen, W)
    return {
        "value": round(cand / dt, 1),
        "unit": "candidate tokens/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"one whole step ({cand} candidates over the three prune steps): fp64 scores, top-k and the "
                  f"gather of all 28 layers' K/V, hidden states and positions; best of {repeats} runs "
                  f"({', '.join(f'{t:.1f}' for t in times)} s) with {threads} BLAS threads on "
                  f"{os.cpu_count()} host CPUs",
        "host_cpus": os.cpu_count(),
        "blas_threads": threads,
        "single_thread_configs_1_3": single,
    }


def single_thread_configs(OP, widen, W, repeats=3):
    """The oracle's prune + compaction of configs 1-3 with one BLAS thread,
    best of `repeats` (inputs widened from their bits inside the timing)."""
    from threadpoolctl import threadpool_limits
    out = {}
    with threadpool_limits(limits=1):
        for cfg, fn in ((1, W.prune_cfg1), (2, W.prune_cfg2), (3, W.prune_cfg3)):
            case = fn()
            cache = W.cfg_cache(cfg, case)
            sd = [dict(tok_off=s.tok_off, n_tokens=s.n_tokens, q_off=s.q_off, q_len=s.q_len, tags=s.tags(),
                       keep=s.keep, keep_basis=s.keep_basis) for s in case.seqs]
            cand = sum(int((s.tags() != 0).sum()) for s in case.seqs)
            best = float("inf")
            for _ in range(repeats):
                t0 = time.perf_counter()
                _, kept, _, _ = OP.prune_batch(widen(case.q, case.dtype), widen(case.k, case.dtype), sd)
                for x in cache.k_layers + cache.v_layers:
                    OP.compact_rows(x, kept, axis=1)
                OP.compact_rows(cache.hidden, kept, axis=0)
                OP.compact_rows(cache.pos, kept, axis=1)
                best = min(best, time.perf_counter() - t0)
            out[f"cfg{cfg}"] = {"seconds": round(best, 4), "candidate_tokens_per_s": round(cand / best, 1)}
    log("cpu oracle, one thread: " + ", ".join(f"{k} {v['seconds']:.3f} s" for k, v in out.items()))
    return out


if __name__ == "__main__":
    main()
