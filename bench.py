"""Throughput of the ODB window pipeline on one MI355X.

One step = grouping (odb_form_groups) + alignment with coverage check
(odb_align_groups) + padded collation (odb_collate) + exact token-level loss-scaling
weights (odb_loss_weights) of a whole window whose CSR token stream is already resident
in HBM.  Steps run double-buffered on two HIP streams: the grouping, alignment and loss
weights of step i+1 (plan stream) run while the collate of step i (collate stream)
streams its outputs; each step has its own plan buffers, the outputs are shared.  The serial
schedule (one stream, plan then collate) is timed too.  Prints one JSON line:

  value        emitted samples per second (whole job)
  roofline     the collate stage (dominant): algorithmic bytes per odb_collate call /
               its average duration from HIP events on the launch stream, vs 8 TB/s, in
               the two-stream schedule (frac) and in the serial one, where nothing runs
               beside it (alone_frac);
               traffic = HBM bytes per call from the committed rocprofv3 counters
               (profiles/), reported only while the collate source is unchanged;
               copy_ceiling_gbs = a plain 4 GiB device copy, as a practical ceiling;
               mix_copy_gbs = a torch broadcast copy (1 GiB read, 4 GiB written) with the
               collate's 1 : 4 read : write bytes
  cpu_baseline the CPU oracle on the same window, single-threaded on this host: the plan
               of the whole window and the collate of its first ranks until about 20 s,
               extrapolated to the whole window per rank
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def collate_alg_bytes(n, real_tokens, padded, slots):
    # 16 B written per padded element (4 int32 outputs), 4 B read per real token, 12 B
    # per row (its sample's token start and length: the plan's row records, or an
    # emitted id and two CSR offsets), 24 B of slot tables per slot
    return 16 * padded + 4 * real_tokens + 8 * (n + 1) + 4 * n + 24 * slots


def window_plan(p, stream):
    p.form(stream)
    p.align(stream)


def window_weights(p, stream):
    p.loss_weights(stream=stream)


def pipelined_steps(pipes, plan_stream, collate_stream, steps, plan=window_plan, weights=window_weights):
    """`steps` steps, double-buffered over the two pipelines in `pipes` (shared outputs):
    step i plans into pipes[i % 2] on `plan_stream` (`plan`: odb_form_groups +
    odb_align_groups for a window, odb_stream_plan for a streaming iteration) once that
    pipeline's previous collate has finished, computes its loss weights there too (they
    read only the plan), and collates on `collate_stream` once its plan is done.  The plan
    calls synchronise only the plan stream, so while the host waits for step i's plan the
    collate stream is still writing step i-1.  Returns the host seconds of the whole loop
    (both streams drained) and per step the HIP-event milliseconds of odb_collate and of
    the loss weights (the latter beside the previous step's collate)."""
    import torch

    free = [torch.cuda.Event(), torch.cuda.Event()]
    for e in free:
        e.record(collate_stream)
    marks = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        p = pipes[i % 2]
        plan_stream.wait_event(free[i % 2])
        plan(p, plan_stream)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ev[2].record(plan_stream)
        weights(p, plan_stream)
        ev[3].record(plan_stream)
        collate_stream.wait_event(ev[3])
        ev[0].record(collate_stream)
        p.collate(collate_stream)
        ev[1].record(collate_stream)
        free[i % 2].record(collate_stream)
        marks.append(ev)
    torch.cuda.synchronize()
    sec = time.perf_counter() - t0
    return sec, [e[0].elapsed_time(e[1]) for e in marks], [e[2].elapsed_time(e[3]) for e in marks]


def serial_steps(pipe, stream, steps):
    """`steps` window steps on one stream, each planned and then collated.  Returns the host
    seconds of the loop and per step the HIP-event milliseconds of odb_collate, which here
    runs with nothing beside it."""
    import torch

    marks = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        pipe.form(stream)
        pipe.align(stream)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record(stream)
        pipe.collate(stream)
        ev[1].record(stream)
        pipe.loss_weights(stream=stream)
        marks.append(ev)
    torch.cuda.synchronize()
    return time.perf_counter() - t0, [e[0].elapsed_time(e[1]) for e in marks]


def measured_traffic(workload):
    """HBM bytes per odb_collate call from the committed rocprofv3 counter record, if it
    was taken on this workload with the collate source as it is now; otherwise None."""
    import hashlib

    path = os.path.join(ROOT, "profiles", f"collate_traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    src = open(os.path.join(ROOT, rec["source"]), "rb").read()
    if hashlib.sha256(src).hexdigest() != rec["source_sha256"] or rec["workload"] != workload:
        return None
    return rec["traffic_bytes"]


def host_cpu():
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return model, len(os.sched_getaffinity(0))


def mix_copy(dev, gib=1.0, reps=5):
    """torch broadcast copy of a `gib` GiB int32 array into a [4, n] output: 4 bytes read
    for every 16 written, the collate's mix, through a library elementwise kernel."""
    import numpy as np
    import torch

    m = int(gib * (1 << 30)) // 4
    src = torch.ones(m, dtype=torch.int32, device=dev)
    dst = torch.empty((4, m), dtype=torch.int32, device=dev)
    view = src.unsqueeze(0).expand(4, m)
    dst.copy_(view)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for a, b in ev:
        a.record()
        dst.copy_(view)
        b.record()
    torch.cuda.synchronize()
    ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    del src, dst, view
    torch.cuda.empty_cache()
    return 20 * m / (ms * 1e-3) / 1e9


def copy_ceiling(dev, gib=4.0, reps=5):
    """Plain device-to-device copy (torch copy_) of `gib` GiB: bytes read + written / time."""
    import numpy as np
    import torch

    m = int(gib * (1 << 30)) // 4
    src = torch.ones(m, dtype=torch.int32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for a, b in ev:
        a.record()
        dst.copy_(src)
        b.record()
    torch.cuda.synchronize()
    ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    del src, dst
    torch.cuda.empty_cache()
    return 8 * m / (ms * 1e-3) / 1e9


def length_sketch_timing(odb, win, ws, w, dev, reps=5):
    """The ROI screen: a 5,000-id random sketch and the whole window (odb_length_sketch
    synchronises, so each call is timed on the host clock, median of `reps`)."""
    import numpy as np
    import torch

    ids = torch.from_numpy(np.random.default_rng(5).choice(w.n, size=min(5000, w.n), replace=False)
                           .astype(np.int32)).to(dev)

    def timed(fn):
        fn()
        t = []
        for _ in range(reps):
            t0 = time.perf_counter()
            out = fn()
            t.append(time.perf_counter() - t0)
        return out, float(np.median(t)) * 1e3

    s5k, ms5k = timed(lambda: odb.odb_length_sketch(win, ids, ids.numel(), w.budget, ws))
    sw, msw = timed(lambda: odb.odb_length_sketch(win, None, w.n, w.budget, ws))
    return {"cv": s5k["cv"], "short_fraction": s5k["short_fraction"], "high_roi": s5k["high_roi"],
            "sketch_ids": int(ids.numel()), "sketch_ms": ms5k, "window_cv": sw["cv"],
            "window_short_fraction": sw["short_fraction"], "window_ms": msw,
            "window_gbs_incl_sync": 8 * (w.n + 1) / (msw * 1e-3) / 1e9}


STREAM_CONFIG = dict(ranks=64, budget=16384, buffer_size=1024, depth=1024, rate=1024, seed=74)


def stream_plan(sp, stream):
    sp.plan(stream)


def stream_weights(sp, stream):
    sp.loss_weights(stream=stream)


def stream_timing(odb, w, tok_off, tokens, dev, plan_stream, collate_stream, iters=3, pipelined_iters=16):
    """Logical iterations of the unified streaming loop over the window's samples as a
    dataset (odb_stream_plan: every round's fetch, grouping, alignment and emission), each
    followed by the collate of its plan.  Serial (host clock around each synchronising
    call, one pipeline) and two-stream (iteration i+1's plan and loss weights beside
    iteration i's collate, two pipelines sharing the outputs)."""
    import numpy as np
    import torch

    c = STREAM_CONFIG
    perm = torch.from_numpy(np.random.default_rng(c["seed"]).permutation(w.n).astype(np.int32)).to(dev)
    win = odb.DeviceWindow(np.linspace(0, w.n, c["ranks"] + 1).astype(np.int64), tok_off, tokens, None, 0)
    sps = [odb.StreamPipeline(win, perm, c["budget"], buffer_size=c["buffer_size"], depth=c["depth"],
                              rate=np.full(c["ranks"], c["rate"], np.int32)) for _ in range(2)]
    for sp in sps:
        sp.plan()
        sp.collate()
        sp.loss_weights()
        sps[1].outputs = sps[0].outputs
    torch.cuda.synchronize()
    sp = sps[0]
    plan_t, coll_t = [], []
    for _ in range(iters):
        t0 = time.perf_counter()
        info = sp.plan()
        t1 = time.perf_counter()
        sp.collate()
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        plan_t.append(t1 - t0)
        coll_t.append(t2 - t1)
    plan_ms = float(np.median(plan_t)) * 1e3
    coll_ms = float(np.median(coll_t)) * 1e3
    pipelined_steps(sps, plan_stream, collate_stream, 2, plan=stream_plan, weights=stream_weights)
    sec, coll_ev, _ = pipelined_steps(sps, plan_stream, collate_stream, pipelined_iters, plan=stream_plan,
                                      weights=stream_weights)
    for x in sps:
        odb.odb_collate_status(x.ws)
        assert x.info["steps"] == info["steps"] and x.info["padded_elems"] == info["padded_elems"]
    two_ms = sec / pipelined_iters * 1e3
    out = {"config": dict(c, samples=w.n, lengths=w.name),
           "plan_ms": plan_ms, "collate_ms": coll_ms,
           "rounds": info["rounds"], "emit_rounds": info["emit_rounds"], "skip_rounds": info["skip_rounds"],
           "us_per_round": plan_ms * 1e3 / max(info["rounds"], 1), "steps": info["steps"],
           "pad_fraction": info["pad_fraction"], "padded_elems": info["padded_elems"],
           "emitted_views": info["emitted_views"],
           "serial_ms_per_iteration": plan_ms + coll_ms,
           "two_stream_ms_per_iteration": two_ms,
           "two_stream_collate_ms": float(np.mean(coll_ev)),
           "samples_per_s": info["emitted_views"] / (two_ms * 1e-3),
           "serial_samples_per_s": info["emitted_views"] / ((plan_ms + coll_ms) * 1e-3)}
    for x in sps:
        x.outputs = None
    del sps, sp
    torch.cuda.empty_cache()
    return out


def cpu_baseline(w, tokens_dev, min_seconds=20.0, pad_id=0):
    """The oracle, single-threaded, on the same window: its plan of the whole window (every
    rank, the alignment over all W ranks), then its collate rank by rank (each rank's
    token range copied back from the device, not timed) until at least `min_seconds` of
    oracle time; the whole window's time is the plan plus the collated ranks' average
    collate time times W (every rank when the bound allows)."""
    import oracle

    t0 = time.perf_counter()
    p = oracle.plan_window(w)
    t_plan = time.perf_counter() - t0
    t_coll = 0.0
    done = 0
    while done < w.W and t_plan + t_coll < min_seconds:
        r = done
        a, b = int(w.tok_off[w.rank_off[r]]), int(w.tok_off[w.rank_off[r + 1]])
        toks = tokens_dev[a:b].cpu().numpy()
        t0 = time.perf_counter()
        out = p.collate_rank(r, w.tok_off, toks, pad_id)
        t_coll += time.perf_counter() - t0
        done += 1
        del toks, out
    est = t_plan + (t_coll / done * w.W if done else 0.0)
    samples = int(p.info["emitted_samples"])
    toks = int(p.info["real_tokens"])
    model, nproc = host_cpu()
    return {
        "value": samples / est,
        "unit": "samples/s",
        "cores": 1,
        "host": f"{model}, {nproc} cores available",
        "kind": "oracle",
        "sample": f"the oracle's plan of the whole window ({w.W} ranks, {w.n} samples, alignment over all ranks: "
                  f"{t_plan:.1f} s) and its collate of ranks 0-{done - 1} ({t_coll:.1f} s); whole-window time = plan "
                  f"+ average rank collate x {w.W} = {est:.1f} s, single-threaded",
        "tokens_per_s": toks / est,
        "plan_seconds": t_plan,
        "collated_ranks": done,
        "collate_seconds": t_coll,
        "whole_window_seconds": est,
    }


def plan_only(odb, w, win, stream, steps, warmup):
    """Grouping + alignment alone, serial on one stream (host clock around both calls, the
    alignment ending in its synchronisation): the plan's latency per window."""
    import numpy as np

    pipe = odb.Pipeline(win, w.budget, mode=w.mode, quota=w.quota, pad_id=0)
    for _ in range(max(warmup, 1)):
        pipe.form(stream)
        pipe.align(stream)
    t = []
    for _ in range(steps):
        t0 = time.perf_counter()
        pipe.form(stream)
        pipe.align(stream)
        t.append(time.perf_counter() - t0)
    ms = float(np.median(t)) * 1e3
    return {"metric": "plan latency (grouping + alignment) on 1 MI355X", "value": w.n / (ms * 1e-3),
            "unit": "samples/s", "ms_per_plan": ms, "ms_min": float(np.min(t)) * 1e3, "steps": steps,
            "warmup": warmup, "n_gpus": 1, "higher_is_better": True, "dtype": "i32", "data": "synthetic",
            "config": {"workload": w.name, "samples": w.n, "simulated_ranks": w.W, "budget": w.budget,
                       "mode": w.mode, "steps_aligned": int(pipe.info["steps"]),
                       "rounds": int(pipe.info["rounds"]), "groups": int(pipe.groups_per_rank.sum())}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=4)
    ap.add_argument("--workload", default="ln480_w64x262144")
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="oracle time after which the CPU baseline stops collating ranks (the plan of the whole "
                         "window is always timed)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-stream", dest="stream", action="store_false",
                    help="skip the unified-streaming-loop measurement")
    ap.add_argument("--calibrate-copy", type=float, default=0.0, metavar="GIB",
                    help="before the steps, run one plain device copy of GIB GiB (int32 -> int32) as a "
                         "known-size reference for hardware byte counters")
    ap.add_argument("--budget", type=int, default=0,
                    help="padded-token budget in place of the workload's (with --plan-only: e.g. 67108864 takes the "
                         "pointer-jumping path on the largest window)")
    ap.add_argument("--plan-only", action="store_true",
                    help="time grouping + alignment alone (serial, one stream), no collate; prints a plan line")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the simulated ranks of a window are "
              "segments of one launch, there is no multi-GPU path", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2606_19989_amd as odb
    import synth

    wl = synth.WORKLOADS[args.workload]
    t = time.time()
    w = wl.window()
    if args.budget > 0:
        w.budget = args.budget
    log(f"[bench] {wl.name}: W={w.W} n={w.n} tokens={w.total_tokens} budget={w.budget} "
        f"(drawn in {time.time() - t:.1f} s)")
    dev = torch.device("cuda:0")
    torch.cuda.init()
    # the two streams are created before any other stream is used, so the runtime puts
    # them on different hardware queues (streams sharing a queue run one after another)
    plan_stream = torch.cuda.Stream(device=dev)
    collate_stream = torch.cuda.Stream(device=dev)
    tok_off, tokens, ident = synth.device_tensors(w, dev)
    torch.cuda.synchronize()
    win = odb.DeviceWindow(w.rank_off, tok_off, tokens, ident, w.num_identities)
    if args.plan_only:
        print(json.dumps(plan_only(odb, w, win, plan_stream, args.steps, args.warmup)), flush=True)
        return
    pipes = [odb.Pipeline(win, w.budget, mode=w.mode, quota=w.quota, pad_id=0) for _ in range(2)]
    pipe = pipes[0]
    log(f"[bench] inputs resident: {(tok_off.numel() * 8 + tokens.numel() * 4) / 1e9:.1f} GB")

    if args.calibrate_copy > 0:
        m = int(args.calibrate_copy * (1 << 30)) // 4
        src = torch.ones(m, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy: {m * 4} bytes read, {m * 4} bytes written")
        del src, dst
        torch.cuda.empty_cache()
    for p in pipes:
        p.run()
        p.loss_weights(odb.ODB_WEIGHT_TOKEN_EXACT)
        pipes[1].outputs = pipes[0].outputs  # one set of outputs, written step by step
    torch.cuda.synchronize()
    info = dict(pipe.info)
    for p in pipes:
        odb.odb_collate_status(p.ws)
    # warm-up in the timed schedule (the first overlapped step runs slow)
    pipelined_steps(pipes, plan_stream, collate_stream, args.warmup)
    log(f"[bench] {args.warmup} warm-up steps done")

    sec, collate_all, weights_all = pipelined_steps(pipes, plan_stream, collate_stream, args.steps)
    log(f"[bench] timed {args.steps} steps (two streams)")
    for p in pipes:
        assert p.info["steps"] == info["steps"] and p.info["padded_elems"] == info["padded_elems"]
        odb.odb_collate_status(p.ws)
    sec_per_step = sec / args.steps
    collate_ms = float(np.mean(collate_all))
    weights_ms = float(np.mean(weights_all))
    serial_n = min(max(3, args.steps // 2), 20)
    serial_sec, collate_alone = serial_steps(pipe, plan_stream, serial_n)
    serial_sec_per_step = serial_sec / serial_n
    collate_alone_ms = float(np.mean(collate_alone))
    log(f"[bench] serial schedule: {serial_sec_per_step * 1e3:.2f} ms/step, odb_collate alone "
        f"{collate_alone_ms:.3f} ms (beside the next plan {collate_ms:.3f} ms)")

    sketch = length_sketch_timing(odb, win, pipe.ws, w, dev)
    log(f"[bench] length sketch: cv={sketch['cv']:.3f} f_s={sketch['short_fraction']:.3f} "
        f"window {sketch['window_ms']:.3f} ms")
    if args.stream:
        # the window pipeline's 129 GB of outputs and the streaming plan's would not both
        # fit in 288 GB
        for p in pipes:
            p.outputs = None
        torch.cuda.empty_cache()
        stream = stream_timing(odb, w, tok_off, tokens, dev, plan_stream, collate_stream)
        log(f"[bench] streaming iteration: plan {stream['plan_ms']:.1f} ms over {stream['rounds']} rounds, "
            f"collate {stream['collate_ms']:.1f} ms; two streams {stream['two_stream_ms_per_iteration']:.1f} ms "
            f"per iteration")
    copy_gbs = copy_ceiling(dev)
    mix_gbs = mix_copy(dev)
    log(f"[bench] plain 4 GiB device copy: {copy_gbs:.0f} GB/s; broadcast copy at the collate's 1:4 mix: "
        f"{mix_gbs:.0f} GB/s")

    n = w.n
    K = pipe.num_slots
    P = int(info["padded_elems"])
    real = int(info["real_tokens"])
    emitted = int(info["emitted_samples"])
    alg = collate_alg_bytes(n, real, P, K)
    achieved = alg / (collate_ms * 1e-3) / 1e9
    result = {
        "metric": "samples/s and tokens/s batched+collated on 1 MI355X; % of HBM peak",
        "value": emitted / sec_per_step,
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": sec_per_step * 1e3,
        "serial_ms_per_step": serial_sec_per_step * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i32",
        "data": "synthetic",
        "tokens_per_s": real / sec_per_step,
        "padded_elems_per_s": P / sec_per_step,
        "pipeline_hbm_frac": alg / sec_per_step / 1e9 / HBM_PEAK_GBS,
        "loss_weights_ms": weights_ms,
        "second_gather_rounds": int(info["second_gather_rounds"]),
        "length_sketch": sketch,
        "stream": stream if args.stream else None,
        "config": {
            "workload": wl.name,
            "description": wl.description,
            "simulated_ranks": w.W,
            "samples": n,
            "real_tokens": real,
            "padded_elems": P,
            "steps_aligned": int(info["steps"]),
            "budget": w.budget,
            "mode": w.mode,
            "pad_fraction": info["pad_fraction"],
            "schedule": "two HIP streams, double-buffered plans: grouping + alignment + loss weights "
                        "of step i+1 run beside the collate of step i",
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "odb_collate (collate_kernel, row records from the plan)",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": measured_traffic(wl.name),
            "alg_bytes_per_launch": alg,
            "avg_launch_ms": collate_ms,
            "median_launch_ms": float(np.median(collate_all)),
            "alone_avg_launch_ms": collate_alone_ms,
            "alone_frac": alg / (collate_alone_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "copy_ceiling_gbs": copy_gbs,
            "mix_copy_gbs": mix_gbs,
        },
    }
    if not args.no_cpu_baseline:
        log(f"[bench] CPU oracle: plan of the whole window, then its collate rank by rank for >= {args.cpu_seconds:.0f} s ...")
        result["cpu_baseline"] = cpu_baseline(w, tokens, min_seconds=args.cpu_seconds)
        log("[bench] CPU oracle done")
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
