"""Benchmark: one training step of one GPU's shard of the pooled embedding layer.

A step is the whole hot path over one fresh seeded batch: pooled forward,
id dedup (sort + unique), gradient segment-reduce fused with the row-wise
Adagrad / SGD update.  Inputs (tables, optimizer state, all batches and
upstream gradients) are resident in HBM before the timed region starts.

Prints ONE JSON line.  `value` is pooled lookups per second of the K timed
steps, run back to back (wall clock; `step_us.timed_region_gpu_per_step` is
one HIP event pair around all of them on the launch stream).  The default
schedule is pipelined: the dedups of the next group of batches run on a side
stream while the main stream runs the forward and update of the current
group (results identical to serial steps bit for bit).  After the timed
region the workspaces' status is read: a step that failed on the device
ends the run with exit status 3.  The same batches then run again as serial
steps with an event pair around each step (`step_us`: median, p10, p90) and
with events between the phases: `roofline` prices the phase that takes the
most time against HBM bandwidth and `phases` lists all three; `cold` repeats
them after flushing the caches.  `cpu_baseline` is the CPU oracle timed on
this host on a bounded sample of the same workload, on all its cores and on
one.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "pooled lookups/sec (fwd+bwd+update) and achieved HBM GB/s vs peak, 1 GPU"
COUNTERS = os.path.join(ROOT, "profiles", "c3_step_hbm_counters.txt")
_CSRC = os.path.join(ROOT, "paper_2112_02752_amd", "csrc")
PHASE_SOURCES = {"fwd": [os.path.join(_CSRC, "pool_fwd.hip")],
                 "dedup": [os.path.join(_CSRC, "dedup.hip"), os.path.join(_CSRC, "emb_common.h")],
                 "bwd_update": [os.path.join(_CSRC, "reduce.hip"), os.path.join(_CSRC, "emb_common.h")]}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=60,
                    help="untimed steps first, each on a batch of its own (the pipelined schedule needs "
                         "several groups of them to reach its steady state)")
    ap.add_argument("--workload", default="c3")
    ap.add_argument("--bags", type=int, default=None, help="bags per table instead of the workload's own")
    ap.add_argument("--opt", choices=("sgd", "adagrad", "adagrad_ew"), default=None,
                    help="optimizer instead of the workload's own (adagrad_ew: element-wise, state [R][D])")
    ap.add_argument("--schedule", choices=("pipelined", "auto", "serial", "concurrent", "stale"),
                    default="pipelined",
                    help="pipelined: the dedups of the next group of batches on side streams while the main "
                         "stream runs the forward and update of the current group; concurrent: the forward of a "
                         "batch on a side stream at the same time as its id dedup; serial: forward, dedup, "
                         "reduce + update one after another on one stream; auto: concurrent for batches of at "
                         "least a million lookups, else serial; stale: the asynchronous schedule with "
                         "staleness one (the forward of batch k+1 on a side stream, reading the table before "
                         "the update of batch k, alongside the dedup of batch k)")
    ap.add_argument("--group", type=int, default=None,
                    help="batches per group of the pipelined schedule (default: the binding's choice for the "
                         "batch size, emb.pipeline_group)")
    ap.add_argument("--depth", type=int, default=2,
                    help="pipelined: buffer set parities (groups whose dedup buffers are in use at once; with 3 "
                         "a chained call's look-ahead dedups need not wait for its last-but-one group)")
    ap.add_argument("--look", type=int, default=1,
                    help="pipelined, chained: groups each call dedups ahead for the next (1..depth-1)")
    ap.add_argument("--no-chain", action="store_true",
                    help="pipelined: time one call on its own (its first group's dedups and its last group's "
                         "forward and update not overlapped) instead of a call in a chain of calls")
    ap.add_argument("--side-streams", type=int, default=3,
                    help="side streams of the pipelined schedule with --dedup per-batch (more than one: the "
                         "dedups of a group run concurrently with emb_unique_ids_concurrent)")
    ap.add_argument("--dedup", choices=("group", "per-batch"), default="group",
                    help="pipelined schedule: each group's dedups as one emb_unique_ids_batched call on one side "
                         "stream (group), or one dedup per batch on the side streams (per-batch)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-cold", action="store_true", help="skip the cold-cache repeat (for counter runs)")
    ap.add_argument("--no-graph", action="store_true", help="skip the HIP-graph replay timing")
    ap.add_argument("--counters-run", action="store_true",
                    help="only the warm-up, the timed region and the phase timings (the kernels of the timed "
                         "configuration and nothing else, for rocprofv3 counter runs)")
    ap.add_argument("--route-ranks", type=int, default=8,
                    help="also time emb_route_ids of the same batches over this many equal row ranges (0: skip)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="budget of the CPU oracle sample")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of known size (for counter calibration)")
    return ap.parse_args()


def byte_models(w, N: float, U: float):
    """Algorithmic bytes per step of each phase, logical (every lookup's row)
    and compulsory (every distinct row once per phase)."""
    M, D = w.num_bags, w.dim
    sw = 4 if w.dtype == "fp32" else 2
    s_state = {"sgd": 0, "adagrad": 4, "adagrad_ew": 4 * D}[w.opt]
    fwd_fixed = 4 * (M + 1) + 4 * N + 4 * M * D
    fwd_log = fwd_fixed + N * D * sw
    fwd_comp = fwd_fixed + U * D * sw
    dedup = 8 * N + 12 * U + 4
    bwd_fixed = 4 * N + 4 * (U + 1) + 4 * (M + 1) + 4 * U + 2 * U * D * sw + 2 * U * s_state
    bwd_log = bwd_fixed + N * D * 4
    bwd_comp = bwd_fixed + M * D * 4
    return {"fwd": (fwd_log, fwd_comp), "dedup": (dedup, dedup), "bwd_update": (bwd_log, bwd_comp)}


def global_keys(row_offset, B, offsets, indices):
    bag = np.repeat(np.arange(len(offsets) - 1), np.diff(offsets))
    return (np.asarray(row_offset, dtype=np.int64)[bag // B] + indices).astype(np.uint32)


def file_sha(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def counter_traffic(workload: str, dedup_kind: str):
    """HBM bytes per step of each phase from the committed rocprofv3 counter
    summary (FETCH_SIZE and WRITE_SIZE scaled by the copy-kernel calibration);
    None for every phase of another workload than the one the counters were
    taken on, for the dedup phase of another dedup than theirs (one call per
    batch, or batched calls over groups of K), and for a phase whose kernel
    sources changed since."""
    if not os.path.exists(COUNTERS):
        return None
    kv = {}
    measured_on = dedup_on = None
    for line in open(COUNTERS):
        if line.startswith("Workload: "):
            measured_on = line[len("Workload: "):].strip()
        if line.startswith("Dedup: "):
            dedup_on = line[len("Dedup: "):].strip()
        if "=" in line and not line.startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    if measured_on != workload:
        return {phase: None for phase in PHASE_SOURCES}
    out = {}
    for phase, src in PHASE_SOURCES.items():
        try:
            ok = all(kv.get(f"sha_{os.path.basename(f)}") == file_sha(f) for f in src)
            ok = ok and (phase != "dedup" or dedup_on == dedup_kind)
            out[phase] = float(kv[f"hbm_bytes_{phase}"]) if ok else None
        except (KeyError, ValueError):
            out[phase] = None
    return out


def copy_calibration():
    import torch
    n = 1 << 28  # 1 GiB of fp32
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n, "launches": 3}), flush=True)


def _oracle_rate(w, batches, budget_s: float):
    """Oracle whole steps on the benchmark's batches, then further seeded
    batches of the same workload, until about `budget_s` seconds of oracle
    time: (lookups per second, steps, lookups, seconds)."""
    import oracle
    import synth
    done_n, elapsed, steps, s = 0, 0.0, 0, 0
    while elapsed < budget_s and s < 400:
        b = batches[s] if s < len(batches) else synth.make_batch(w, s)
        keys = np.unique(global_keys(w.row_offset, w.bags_per_table, b.offsets, b.indices))
        store = oracle.RowStore(synth.weight_rows(w, keys), keys=keys,
                                state=np.zeros(len(keys), np.float32) if w.opt == "adagrad" else None)
        t0 = time.perf_counter()
        oracle.step(w.num_tables, w.row_offset, w.bags_per_table, b.offsets, b.indices, b.grad, store, w.pool,
                    w.opt, w.lr, w.eps)
        elapsed += time.perf_counter() - t0
        done_n += len(b.indices)
        steps += 1
        s += 1
    return done_n / elapsed, steps, done_n, elapsed


def cpu_baseline(w, batches, budget_s: float):
    """The oracle, untuned, on whole steps of the same workload: on all the
    host's cores (its loops over bags and segments in parallel, the sort on
    one thread; the results do not depend on the thread count), then on one."""
    import oracle
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or (os.cpu_count() or 1)
    what = (f"whole steps of {w.name} (fwd+dedup+reduce+update; the rows a batch touches regenerated from the "
            f"seed, untimed)")
    try:
        oracle.set_threads(threads)
        used = oracle.get_threads()
        rate, steps, n, t = _oracle_rate(w, batches, budget_s)
        oracle.set_threads(1)
        rate1, steps1, n1, t1 = _oracle_rate(w, batches, budget_s)
    finally:
        oracle.set_threads(0)
    return {"value": rate, "unit": "lookups/s", "cores": used, "kind": "oracle",
            "sample": f"{steps} {what}, {n} lookups, {t:.1f} s of oracle time on {used} threads",
            "single_thread": {"value": rate1, "unit": "lookups/s", "cores": 1,
                              "sample": f"{steps1} {what}, {n1} lookups, {t1:.1f} s of oracle time"},
            "host": {"cpu_model": host_cpu_model(), "nproc": os.cpu_count(),
                     "omp_num_threads": os.environ.get("OMP_NUM_THREADS")}}


def host_cpu_model() -> str:
    """The host CPU's model name (the oracle's machine), from /proc/cpuinfo."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cost_model_check(w, N, U, t_phase, serial_step_s=None):
    """The layer's cost model (fitted to earlier MI355X measurements of serial
    steps: one emb_unique_ids call per batch) next to this run's measured
    phase times.  With serial_step_s (the phases were timed with group
    dedups, which the model does not describe) the dedup is left out and the
    step is compared with the median serial step instead."""
    from paper_2112_02752_amd import cost
    pr = cost.predict(N, U, w.total_rows, w.dim, w.dtype, w.opt)
    meas = {k: v * 1e6 for k, v in t_phase.items()}
    if serial_step_s is None:
        meas["step"] = sum(meas.values())
        note = "measured: this run's phase timings, serial steps"
    else:
        meas.pop("dedup")
        meas["step"] = serial_step_s * 1e6
        note = ("measured: this run's phase timings, whose dedup (emb_unique_ids_batched) the model does not "
                "describe, and the median serial step (one emb_unique_ids call per step)")
    return {"predicted_us": {k: round(v, 2) for k, v in pr.items()},
            "measured_us": {k: round(v, 2) for k, v in meas.items()},
            "rel_err": {k: round((pr[k] - meas[k]) / meas[k], 4) for k in meas}, "note": note}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: this build measures one GPU's shard of the embedding layer; "
              "multi-GPU runs are not part of it", file=sys.stderr)
        sys.exit(2)
    import torch
    import synth
    import paper_2112_02752_amd as emb

    if args.copy_calibration:
        copy_calibration()
        return

    w = synth.workload(args.workload)
    if args.opt is not None and args.opt != w.opt:
        import dataclasses
        w = dataclasses.replace(w, opt=args.opt, name=f"{w.name}-{args.opt}",
                                description=f"{w.description}; optimizer {args.opt} instead")
    if args.bags is not None and args.bags != w.bags_per_table:
        import dataclasses
        w = dataclasses.replace(w, bags_per_table=args.bags, name=f"{w.name}-b{args.bags}",
                                description=f"{w.description}; {args.bags} bags per table instead")
    dev = "cuda"
    # every step, warm-up or timed, gets a batch of its own: the warm-up
    # steps touch as much of the table as steady-state training has touched
    # recently (with fewer distinct warm-up batches the first timed steps
    # run slower)
    n_warm = args.warmup
    t0_batch = n_warm
    total = n_warm + args.steps
    # the stale schedule's last timed step runs the forward of one more batch;
    # the chained pipelined schedule's timed call dedups the groups after its
    # steps (`look` of them, below depth and as many as its steps hold), and its own first
    # groups are deduplicated at the end of the warm-up: the timed region
    # holds exactly `steps` dedups and `steps` forwards, backwards and
    # updates.  The pipelined schedule also runs one call on its own over
    # `steps` batches of their own (isolated_call).
    print(f"[bench] {w.name}: {w.description}", file=sys.stderr, flush=True)
    t0 = time.time()
    first = synth.make_batch(w, 0)
    group = args.group if args.group else emb.pipeline_group(len(first.indices))
    look = min(args.look, args.depth - 1, args.steps // group) if args.schedule == "pipelined" else 0
    chain = args.schedule == "pipelined" and not args.no_chain and look > 0
    n_ahead = look * group if chain else 0
    n_iso = args.steps if args.schedule == "pipelined" else 0
    n_batches = total + (1 if args.schedule == "stale" else 0) + n_ahead + n_iso
    batches = [first] + [synth.make_batch(w, s) for s in range(1, n_batches)]
    print(f"[bench] generated {n_batches} batches in {time.time() - t0:.1f} s", file=sys.stderr, flush=True)
    W = torch.empty((w.total_rows, w.dim), dtype=torch.float32 if w.dtype == "fp32" else torch.bfloat16,
                    device=dev)
    synth.fill_device_weights(w, W.data_ptr(), int(torch.cuda.current_stream().cuda_stream))
    state = None
    if w.opt == "adagrad":
        state = torch.zeros(w.total_rows, dtype=torch.float32, device=dev)
    elif w.opt == "adagrad_ew":
        state = torch.zeros((w.total_rows, w.dim), dtype=torch.float32, device=dev)
    tables = emb.Tables(W, [int(x) for x in w.row_offset])
    nmax = max(len(b.indices) for b in batches)
    layer = emb.Layer(tables, w.pool, w.opt, w.lr, w.eps, state, max_indices=nmax, max_bags=w.num_bags)
    dev_batches = []
    for b in batches:
        off = torch.from_numpy(b.offsets).to(dev)
        idx = torch.from_numpy(b.indices).to(dev)
        g = torch.from_numpy(b.grad).to(dev)
        dev_batches.append((emb.Batch(off, idx, w.bags_per_table), g, len(b.indices)))
    out = torch.empty((w.num_bags, w.dim), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    sp = int(stream.cuda_stream)
    torch.cuda.synchronize()

    def step(i, ev=None):
        b, g, _ = dev_batches[i]
        if ev:
            ev[0].record(stream)
        emb.pool_fwd(tables, b, w.pool, out, sp)
        if ev:
            ev[1].record(stream)
        emb.unique_ids(tables, b, layer.unique_keys, layer.counts, layer.seg_offsets, layer.sort_perm,
                       layer.num_unique, layer.ws, sp)
        if ev:
            ev[2].record(stream)
        emb.grad_reduce(tables, b, w.pool, g, layer.sort_perm, layer.seg_offsets, layer.unique_keys,
                        layer.num_unique, layer.ws, opt=w.opt, lr=w.lr, eps=w.eps, state=state, stream=sp)
        if ev:
            ev[3].record(stream)

    clayer = pipe = None
    if args.schedule in ("concurrent", "auto"):
        clayer = emb.Layer(tables, w.pool, w.opt, w.lr, w.eps, state, max_indices=nmax, max_bags=w.num_bags,
                           concurrent=True if args.schedule == "concurrent" else "auto")

        def run_steps(idx):
            for i in idx:
                clayer.step(dev_batches[i][0], out, dev_batches[i][1], sp)
    elif args.schedule == "pipelined":
        pipe = emb.Pipeline(tables, w.pool, w.opt, w.lr, w.eps, state, max_indices=nmax, max_bags=w.num_bags,
                            group=group, side_streams=args.side_streams, group_dedup=args.dedup == "group",
                            depth=args.depth)

        def run_steps(idx, ahead=None):
            pipe.run([(dev_batches[i][0], out, dev_batches[i][1]) for i in idx], sp,
                     ahead=[dev_batches[i][0] for i in ahead] if ahead else None)
    elif args.schedule == "stale":
        clayer = emb.Layer(tables, w.pool, w.opt, w.lr, w.eps, state, max_indices=nmax, max_bags=w.num_bags,
                           concurrent=True)

        def run_steps(idx):
            # step i: the forward of batch i + 1 (stale by the update of batch
            # i) and the backward + update of batch i.  The warm-up starts with
            # the forward of batch 0 and ends with that of the first timed
            # batch, so every timed step is one whole forward and one whole
            # backward + update.
            idx = list(idx)
            if idx and idx[0] == 0:
                clayer.forward(dev_batches[0][0], out, sp)
            for i in idx:
                clayer.step_stale(dev_batches[i + 1][0], out, dev_batches[i][0], dev_batches[i][1], sp)
    else:
        def run_steps(idx):
            for i in idx:
                layer.step(dev_batches[i][0], out, dev_batches[i][1], sp)

    def check_status(where):
        """A step that failed on the device (a bounded wait of its dedup ran
        out) wrote no table row: its time would not be a step's, so the run
        ends here with the reason."""
        try:
            for obj in (layer, clayer, pipe):
                if obj is not None:
                    obj.check(sp)
        except emb.StepFailed as e:
            print(f"bench.py: {where}: {e}", file=sys.stderr, flush=True)
            sys.exit(3)

    if chain and n_warm > 0:
        run_steps(range(n_warm), ahead=range(t0_batch, t0_batch + n_ahead))
    else:
        run_steps(range(n_warm))
    torch.cuda.synchronize()
    check_status("warm-up")

    # timed region: K whole steps back to back, one fresh batch each, one HIP
    # event pair around all of them on the launch stream
    e_all = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    e_all[0].record(stream)
    if chain:
        run_steps(range(t0_batch, total), ahead=range(total, total + n_ahead))
    else:
        run_steps(range(t0_batch, total))
    e_all[1].record(stream)
    t_enq = time.perf_counter() - t_start
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    gpu_all_s = e_all[0].elapsed_time(e_all[1]) * 1e-3
    check_status("timed region")
    isolated = None
    if n_iso and not args.counters_run:
        # the same schedule as one call on its own over batches of its own
        pipe.discard()
        iso = range(total + n_ahead, total + n_ahead + n_iso)
        torch.cuda.synchronize()
        t_iso = time.perf_counter()
        run_steps(iso)
        torch.cuda.synchronize()
        t_iso = time.perf_counter() - t_iso
        check_status("isolated call")
        isolated = {"us_per_step": t_iso / n_iso * 1e6,
                    "lookups_per_s": sum(dev_batches[i][2] for i in iso) / t_iso,
                    "note": "one pipelined call on its own over `steps` batches of their own, after the timed "
                            "region: its first group's dedups and its last group's forward and update overlap "
                            "nothing"}

    # the same batches again as serial steps with an event pair around each
    # step: the distribution of serial step times
    step_s = None
    if not args.counters_run:
        sev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
        for k, i in enumerate(range(t0_batch, total)):
            sev[k][0].record(stream)
            layer.step(dev_batches[i][0], out, dev_batches[i][1], sp)
            sev[k][1].record(stream)
        torch.cuda.synchronize()
        step_s = [e[0].elapsed_time(e[1]) * 1e-3 for e in sev]

    # per-phase times for the roofline: the same batches again, one phase at a
    # time with events between, through the kernels of the timed
    # configuration.  With group dedups (the pipelined schedule's default)
    # each group's dedups are one batched call and a batch's dedup time is its
    # group's over the group's size; otherwise serial steps.
    group_phases = pipe is not None and pipe.group_ws is not None
    ph = {"fwd": [], "dedup": [], "bwd_update": []}
    torch.cuda.synchronize()
    if group_phases:
        pipe.discard()
        idx = list(range(t0_batch, total))
        recs = []
        for g0 in range(0, len(idx), pipe.K):
            grp = idx[g0:g0 + pipe.K]
            # the device spins while the host enqueues the group (a batched
            # dedup and two calls per batch take the host longer than the
            # device), so that the events time the kernels and not the host:
            # about 0.2 ms of spin per batch, several times the host's time
            if hasattr(torch.cuda, "_sleep"):
                torch.cuda._sleep((1 << 19) * len(grp))
            eg = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            eg[0].record(stream)
            emb.unique_ids_batched(tables, [dev_batches[i][0] for i in grp], pipe.sets[:len(grp)], pipe.group_ws,
                                   sp)
            eg[1].record(stream)
            es = []
            for j, i in enumerate(grp):
                d = pipe.sets[j]
                e3 = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
                e3[0].record(stream)
                emb.pool_fwd(tables, dev_batches[i][0], w.pool, out, sp)
                e3[1].record(stream)
                emb.grad_reduce(tables, dev_batches[i][0], w.pool, dev_batches[i][1], d.sort_perm, d.seg_offsets,
                                d.unique_keys, d.num_unique, d.ws, opt=w.opt, lr=w.lr, eps=w.eps, state=state,
                                stream=sp)
                e3[2].record(stream)
                es.append(e3)
            recs.append((eg, es))
        torch.cuda.synchronize()
        check_status("phase timings")
        for eg, es in recs:
            dd = eg[0].elapsed_time(eg[1]) * 1e-3 / len(es)
            for e3 in es:
                ph["fwd"].append(e3[0].elapsed_time(e3[1]) * 1e-3)
                ph["dedup"].append(dd)
                ph["bwd_update"].append(e3[1].elapsed_time(e3[2]) * 1e-3)
    else:
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
        for k, i in enumerate(range(t0_batch, total)):
            step(i, evs[k])
        torch.cuda.synchronize()
        for e in evs:
            ph["fwd"].append(e[0].elapsed_time(e[1]) * 1e-3)
            ph["dedup"].append(e[1].elapsed_time(e[2]) * 1e-3)
            ph["bwd_update"].append(e[2].elapsed_time(e[3]) * 1e-3)
    phased_step_s = [a + b + c for a, b, c in zip(ph["fwd"], ph["dedup"], ph["bwd_update"])]

    # cold steps: the same batches again, with the L2s and the last-level
    # cache flushed by writing 1 GiB before each step (outside the events)
    flush = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    cold = None
    if not args.no_cold and not args.counters_run:
        cold_evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
        for k, i in enumerate(range(t0_batch, total)):
            flush.fill_(k & 0xff)
            step(i, cold_evs[k])
        torch.cuda.synchronize()
        cold_step_s = [e[0].elapsed_time(e[3]) * 1e-3 for e in cold_evs]
        cold_ph = {"fwd": [e[0].elapsed_time(e[1]) * 1e-3 for e in cold_evs],
                   "dedup": [e[1].elapsed_time(e[2]) * 1e-3 for e in cold_evs],
                   "bwd_update": [e[2].elapsed_time(e[3]) * 1e-3 for e in cold_evs]}
        cold = {"note": "serial steps of the same batches again, 1 GiB written between steps to flush L2 and the "
                        "last-level cache",
                "median_us": float(np.median(cold_step_s)) * 1e6,
                "p10_us": float(np.percentile(cold_step_s, 10)) * 1e6,
                "p90_us": float(np.percentile(cold_step_s, 90)) * 1e6,
                "phases_median_us": {k: float(np.median(v)) * 1e6 for k, v in cold_ph.items()}}
    # achievable streaming bandwidth on this device: a 1 GiB device-to-device copy (read + write)
    dst = torch.empty_like(flush)
    dst.copy_(flush)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    c0.record(stream)
    for _ in range(5):
        dst.copy_(flush)
    c1.record(stream)
    torch.cuda.synchronize()
    copy_gbs = 5 * 2 * (1 << 30) / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del flush, dst

    # routing of the same batches to the owners of equal row ranges: the step
    # before the forward when the table is sharded over that many devices
    routing = None
    if args.route_ranks > 0 and not args.counters_run:
        Wr = args.route_ranks
        shard = [w.total_rows * r // Wr for r in range(Wr + 1)]
        i32 = dict(dtype=torch.int32, device=dev)
        rcnt = torch.empty(Wr, **i32)
        rids, rpos, rbag = (torch.empty(nmax, **i32) for _ in range(3))
        rws = torch.empty(emb.route_workspace_size(nmax, w.num_bags, Wr), dtype=torch.uint8, device=dev)
        for i in range(n_warm):
            emb.route_ids(tables, dev_batches[i][0], shard, rcnt, rids, rpos, rbag, rws, sp)
        rev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
        torch.cuda.synchronize()
        for k, i in enumerate(range(t0_batch, total)):
            rev[k][0].record(stream)
            emb.route_ids(tables, dev_batches[i][0], shard, rcnt, rids, rpos, rbag, rws, sp)
            rev[k][1].record(stream)
        torch.cuda.synchronize()
        r_s = float(np.median([e[0].elapsed_time(e[1]) * 1e-3 for e in rev]))
        r_bytes = 4 * (w.num_bags + 1) + 4 * np.mean([dev_batches[i][2] for i in range(t0_batch, total)]) * 4 \
            + 4 * Wr
        routing = {"ranks": Wr, "shard": "equal row ranges", "kernels": "k_route_count, k_route_scan, "
                   "k_route_scatter (emb_route_ids)", "median_us": r_s * 1e6,
                   "ids_per_s": float(np.mean([dev_batches[i][2] for i in range(t0_batch, total)])) / r_s,
                   "bytes_per_launch": float(r_bytes), "achieved_GBs": r_bytes / r_s / 1e9,
                   "frac": r_bytes / r_s / 1e9 / HBM_PEAK_GBS}

    # the serial step captured in a HIP graph: one batch, replayed back to back,
    # against the same batch's eager steps (the step launches only kernels)
    graph = None
    if not args.no_graph and not args.counters_run:
        i0 = t0_batch
        reps = 20
        ge = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        torch.cuda.synchronize()
        ge[0].record(stream)
        for _ in range(reps):
            layer.step(dev_batches[i0][0], out, dev_batches[i0][1], sp)
        ge[1].record(stream)
        torch.cuda.synchronize()
        try:
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr):
                layer.step(dev_batches[i0][0], out, dev_batches[i0][1])
            gr.replay()
            torch.cuda.synchronize()
            ge[2].record(stream)
            for _ in range(reps):
                gr.replay()
            ge[3].record(stream)
            torch.cuda.synchronize()
            graph = {"note": f"serial steps of batch {i0} ({dev_batches[i0][2]} lookups), {reps} back to back "
                             f"each way", "eager_us_per_step": ge[0].elapsed_time(ge[1]) * 1e3 / reps,
                     "graph_replay_us_per_step": ge[2].elapsed_time(ge[3]) * 1e3 / reps}
            del gr
        except RuntimeError as e:  # reported, not fatal: the headline does not depend on it
            graph = {"error": str(e)[:200]}

    check_status("after the serial, phase-timed and cold steps")
    n_lookups = sum(dev_batches[i][2] for i in range(t0_batch, total))

    # unique counts of the timed batches (for the byte models)
    us = []
    for i in range(t0_batch, total):
        b = batches[i]
        us.append(len(np.unique(global_keys(w.row_offset, w.bags_per_table, b.offsets, b.indices))))
    N_avg = n_lookups / args.steps
    U_avg = float(np.mean(us))
    models = byte_models(w, N_avg, U_avg)
    t_phase = {k: float(np.mean(v)) for k, v in ph.items()}
    dedup_kind = f"emb_unique_ids_batched, groups of {pipe.K}" if group_phases else "emb_unique_ids"
    traffic = counter_traffic(f"{w.name}: {w.description}", dedup_kind)
    dedup_kernels = ("per group of batches: k_prepare_group, then per pass k_tile_counts + k_column_scan + "
                     "k_sort_pass (the last writing each batch's share into its own buffers), then "
                     "k_uniq_counts_group, k_uniq_scan_group, k_unique_group "
                     f"(emb_unique_ids_batched over groups of {pipe.K}; per batch: the group's time over its "
                     "size)") if group_phases else "k_sort_pass x passes + k_unique (emb_unique_ids)"
    phases = {}
    for name, kern in (("fwd", "k_pool_fwd (emb_pool_fwd)"),
                       ("dedup", dedup_kernels),
                       ("bwd_update", "k_reduce_main + k_reduce_combine (emb_grad_reduce, fused update)")):
        log_b, comp_b = models[name]
        t = t_phase[name]
        phases[name] = {"kernels": kern, "avg_us": t * 1e6, "logical_bytes": log_b, "compulsory_bytes": comp_b,
                        "logical_frac": log_b / t / 1e9 / HBM_PEAK_GBS,
                        "compulsory_frac": comp_b / t / 1e9 / HBM_PEAK_GBS,
                        "hbm_traffic_bytes": traffic.get(name) if traffic else None}
    dom = max(phases, key=lambda k: phases[k]["avg_us"])
    d = phases[dom]
    achieved = d["logical_bytes"] / (d["avg_us"] * 1e-6) / 1e9
    step_log = sum(v[0] for v in models.values())
    step_comp = sum(v[1] for v in models.values())
    ms = elapsed / args.steps * 1e3
    line = {
        "metric": METRIC, "value": n_lookups / elapsed, "unit": "lookups/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32" if w.dtype == "fp32" else "bf16 tables, f32 accumulate",
        "data": "synthetic (seeded Zipf ids, N(0,1) upstream gradients, U(-0.01,0.01) tables)",
        "config": {"workload": f"{w.name}: {w.description}", "rows": w.total_rows, "dim": w.dim,
                   "bags": w.num_bags, "lookups_per_step": N_avg, "unique_rows_per_step": U_avg,
                   "table_bytes": w.weight_bytes, "schedule": args.schedule,
                   "staleness": 1 if args.schedule == "stale" else 0,
                   "group": group if args.schedule == "pipelined" else None,
                   "chained": chain,
                   "depth": args.depth if args.schedule == "pipelined" else None,
                   "look_ahead_groups": look if chain else 0,
                   "step_accounting": ("chained calls (a training loop's look-ahead): the warm-up call ends with "
                                       "the dedups of the first timed groups, the timed call with those of the "
                                       "groups after it; the timed region holds exactly `steps` dedups and "
                                       "`steps` forwards, backwards and updates") if chain else None,
                   "dedup": args.dedup if args.schedule == "pipelined" else None,
                   "side_streams": (pipe.S if pipe is not None else None),
                   "overlapped_steps": args.steps if args.schedule == "pipelined" else
                   sum(1 for i in range(t0_batch, total)
                       if clayer is not None and clayer.overlaps(dev_batches[i][2]))},
        "roofline": {"bound": "hbm", "phase": dom, "kernel": d["kernels"], "model": "logical",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": d["hbm_traffic_bytes"], "bytes_per_launch": d["logical_bytes"],
                     "avg_launch_us": d["avg_us"]},
        "phases": phases,
        "step_bytes": {"logical": step_log, "compulsory": step_comp,
                       "logical_GBs": step_log / (ms * 1e-3) / 1e9,
                       "compulsory_GBs": step_comp / (ms * 1e-3) / 1e9,
                       "logical_frac": step_log / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS},
        "step_us": {"schedule": args.schedule, "timed_region_gpu_per_step": gpu_all_s / args.steps * 1e6,
                    "serial_note": "mean / median / p10 / p90: serial steps of the same batches, one event pair "
                                   "around each",
                    "mean": float(np.mean(step_s)) * 1e6 if step_s else None,
                    "median": float(np.median(step_s)) * 1e6 if step_s else None,
                    "p10": float(np.percentile(step_s, 10)) * 1e6 if step_s else None,
                    "p90": float(np.percentile(step_s, 90)) * 1e6 if step_s else None,
                    "host_enqueue_us": t_enq / args.steps * 1e6,
                    "with_phase_events_median": float(np.median(phased_step_s)) * 1e6},
        "isolated_call": isolated,
        "cold": None if cold is None else dict(cold, lookups_per_s=N_avg * 1e6 / cold["median_us"]),
        "achievable_copy_GBs": copy_gbs,
        "routing": routing,
        "graph": graph,
        "cost_model": cost_model_check(w, N_avg, U_avg, t_phase,
                                       float(np.median(step_s)) if group_phases and step_s else None),
    }
    if not args.no_cpu_baseline and not args.counters_run:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(w, batches, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
