"""Benchmark one sparse-embedding training step on one MI355X.

A step is the whole hot path on one synthetic batch: tc_embed_forward_cast
(the forward gather-reduce and Tensor Casting in one call, overlapped), then
tc_embed_backward_update (the casted backward and the sparse update in one
pass), back to back on one stream, with inputs already resident in HBM.
--no-overlap calls tc_embed_forward and tc_cast_index instead of the first;
--unfused makes every step a separate call (tc_embed_forward, tc_cast_index,
tc_embed_backward, tc_sparse_update). Prints ONE JSON line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--config c4] [--also c3,c5,c2,c1]
                  [--no-overlap] [--unfused]

The headline workload (--config, default c4) is the largest one that fits
one GPU: 32 tables x 1M rows x 256 fp32, batch 8192, 20 uniform indices per
bag, SGD. The line also carries compact results (steps/s, per-call times,
HBM fractions, longest segment) for the workloads named by --also, timed
the same way, each after the previous one's memory is freed.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published
NUM_BATCHES = 4        # distinct pre-generated batches the timed steps cycle through


def algorithmic_bytes(w, n, u, nbags):
    """Bytes each call moves under the paper's analytic model (every gather
    counted once, Sec. III-C): index reads, one row read per gather, row
    writes."""
    D4 = 4 * w.dim
    fwd = n * 4 + (nbags + 1) * 4 + n * D4 + nbags * D4
    cast = n * 4 + (nbags + 1) * 4 + n * 4 + u * 4 + (u + 1) * 4
    bwd = n * 4 + (u + 1) * 4 + n * D4 + u * D4
    # G, W in, W out (+ A in, A out: a row of A, or one value per row)
    rows_rw = 5 if w.optimizer in ("adagrad", "rmsprop") else 3
    upd = u * 4 + rows_rw * u * D4 + (8 * u if w.optimizer == "rowwise_adagrad" else 0)
    # fused: the coalesced rows stay in registers (no G written, no G read)
    fused = n * 4 + (u + 1) * 4 + n * D4 + u * 4 + (rows_rw - 1) * u * D4
    return {"forward": fwd, "cast": cast, "backward": bwd, "update": upd,
            "backward_update": fused, "forward_cast": fwd + cast}


def compulsory_bytes(w, n, u, nbags):
    """A lower bound per call: as algorithmic_bytes, but every distinct row a
    call gathers is read once (the forward's U table rows, the backward's
    T*B output-gradient rows), as a perfect cache would give."""
    D4 = 4 * w.dim
    a = algorithmic_bytes(w, n, u, nbags)
    fwd = a["forward"] - n * D4 + u * D4
    bwd_saved = n * D4 - nbags * D4
    return {"forward": fwd, "cast": a["cast"], "backward": a["backward"] - bwd_saved,
            "update": a["update"], "backward_update": a["backward_update"] - bwd_saved,
            "forward_cast": fwd + a["cast"]}


def host_cpu():
    """Model name and usable core count of the host CPU."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = os.cpu_count()
    return {"cpu_model": model, "nproc": usable, "os_cpu_count": os.cpu_count()}


# Sources of each call's kernels, and the kernels one call launches.
KERNEL_SOURCES = {
    "forward": ["tc_internal.h", "tc_group_sum.h", "tc_gather_reduce.hip"],
    "backward": ["tc_internal.h", "tc_group_sum.h", "tc_optim.h", "tc_backward.hip"],
    "backward_update": ["tc_internal.h", "tc_group_sum.h", "tc_optim.h", "tc_backward.hip"],
    "update": ["tc_internal.h", "tc_optim.h", "tc_update.hip"],
    "cast": ["tc_internal.h", "tc_group_sum.h", "tc_cast.hip"],
    "forward_cast": ["tc_internal.h", "tc_group_sum.h", "tc_gather_reduce.hip", "tc_cast.hip"],
}
KERNEL_NAMES = {
    "forward": ["k_forward"],
    # with the backward workspace, as the step runs them
    "backward": ["k_backward_init", "k_backward_short", "k_backward_list"],
    "backward_update": ["k_backward_init", "k_backward_short", "k_backward_list"],
    "update": ["k_sparse_update"],
    "cast": ["k_cast_small", "k_build_keys", "k_radix_hist", "k_radix_scan", "k_radix_scatter",
             "k_seg_count", "k_seg_write"],
    # the forward's bags run in the pair build's launch (or beside k_cast_small)
    "forward_cast": ["k_cast_small", "k_forward_build", "k_radix_hist", "k_radix_scan",
                     "k_radix_scatter", "k_seg_count", "k_seg_write", "k_forward"],
}


def step_calls(args, w):
    """The library calls of one step, in order."""
    rowwise = w.optimizer == "rowwise_adagrad"   # no fused backward + update for it
    first = ["forward", "cast"] if (args.unfused or args.no_overlap) else ["forward_cast"]
    last = ["backward", "update"] if (args.unfused or rowwise) else ["backward_update"]
    return first + last


def source_sha(call: str) -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[call]:
        h.update(open(os.path.join(ROOT, "paper_2010_13100_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def load_traffic(call: str, workload: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel source (else None)."""
    p = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(p):
        return None
    entry = json.load(open(p)).get(f"{call}:{workload}")
    if not entry or entry.get("source_sha") != source_sha(call):
        return None
    return entry["hbm_bytes_per_launch"]


def run_ab(args, w, trainer, dbat, stream):
    """The paper's backward A/B (Sec. VI-A) on this GPU: baseline gradient
    expand-coalesce (expand, stable argsort, Algorithm 1 accumulate) against
    Tensor Casting (cast, Algorithm 3 gather-reduce), same batches, both
    producing the coalesced gradient rows. Each variant's calls of one step
    are bracketed by one event pair; the first `warmup` steps are untimed."""
    import numpy as np
    import torch

    def variant(name, i):
        d = dbat[i % NUM_BATCHES]
        if name == "casted":
            trainer.cast(d["off"], d["idx"], d["bo"], d["n"], stream)
            trainer.backward(d["grad"], stream)
        else:
            trainer.baseline_backward(d["off"], d["idx"], d["bo"], d["n"], d["grad"], stream)

    times = {"baseline": [], "casted": []}
    for i in range(args.warmup + args.steps):
        for name in ("baseline", "casted"):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            variant(name, i)
            e1.record(stream)
            if i >= args.warmup:
                times[name].append((e0, e1))
    torch.cuda.synchronize()
    us = {k: float(np.mean([a.elapsed_time(b) for a, b in v])) * 1e3 for k, v in times.items()}
    uniq = []
    for i in range(NUM_BATCHES):
        d = dbat[i]
        trainer.cast(d["off"], d["idx"], d["bo"], d["n"], stream)
        uniq.append(int(trainer.num_unique.item()))
    D4, nb = 4 * w.dim, w.num_bags
    n = float(np.mean([d["n"] for d in dbat]))
    u = float(np.mean(uniq))
    # paper's traffic model (Sec. III-C): expand reads each bag's gradient and
    # writes N rows; coalesce reads N rows and writes U rows; the casted
    # gather-reduce reads N (gathered) rows and writes U rows
    base_bytes = nb * D4 + n * D4 + n * D4 + u * D4 + 3 * n * 4
    cast_bytes = n * D4 + u * D4 + 2 * n * 4
    return {
        "metric": "backward A/B: baseline expand-coalesce vs Tensor Casting, us per step",
        "config": {"workload": f"{args.config}: {w.name}", "pairs_per_step": round(n, 1),
                   "unique_rows_per_step": round(u, 1)},
        "steps": args.steps, "warmup": args.warmup,
        "baseline_us": round(us["baseline"], 2),
        "casted_us": round(us["casted"], 2),
        "speedup": round(us["baseline"] / us["casted"], 3),
        "algorithmic_bytes": {"baseline": round(base_bytes), "casted": round(cast_bytes),
                              "ratio": round(base_bytes / cast_bytes, 3)},
        "note": "both variants include their sort (argsort / cast); dtype f32; data synthetic",
    }


def write_traffic(pmc_dir: str, workload: str, calls) -> dict:
    """Turn rocprofv3 --pmc CSV runs into HBM bytes per call launch and store
    them in profiles/traffic.json under "<call>:<workload>".

    pmc_dir holds copy_fetch/, copy_write/ (bench.py --copy-calibration runs)
    and fetch/, write/ (runs of `bench.py --profile-steps` on this workload,
    which launch the step's calls and nothing else of the library), each with
    the run_counter_collection.csv that `rocprofv3 --pmc FETCH_SIZE|WRITE_SIZE
    -f csv -o run` writes, plus `steps` (step runs in the profiled program)
    and `copy_bytes`. FETCH_SIZE and WRITE_SIZE are KiB per dispatch; each is
    scaled by copy_bytes / counter-reading-for-the-copy, the counter's own
    error on a plain device copy of known size. A call's bytes per launch
    are the scaled bytes of all dispatches of its kernels over the number of
    steps."""
    import csv
    import re

    def rows(sub):
        with open(os.path.join(pmc_dir, sub, "run_counter_collection.csv")) as f:
            return list(csv.DictReader(f))

    def per_kernel(sub):
        out: dict = {}
        for r in rows(sub):
            out.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]) * 1024.0)
        return out

    scale = {}
    bytes_per_copy = int(open(os.path.join(pmc_dir, "copy_bytes")).read())
    for sub, counter in (("copy_fetch", "FETCH_SIZE"), ("copy_write", "WRITE_SIZE")):
        copies = [float(r["Counter_Value"]) * 1024.0 for r in rows(sub)
                  if "copyBuffer" in r["Kernel_Name"]]
        scale[counter] = bytes_per_copy / (sum(copies) / len(copies))
    steps = int(open(os.path.join(pmc_dir, "steps")).read())
    fetch, write = per_kernel("fetch"), per_kernel("write")
    p = os.path.join(ROOT, "profiles", "traffic.json")
    table = json.load(open(p)) if os.path.exists(p) else {}
    for call in calls:
        fb = wb = 0.0
        seen = []
        for k in KERNEL_NAMES[call]:
            pat = re.compile(r"\b" + k + r"\b")
            fv = [v for n, vs in fetch.items() if pat.search(n) for v in vs]
            wv = [v for n, vs in write.items() if pat.search(n) for v in vs]
            if fv and wv:
                seen.append(k)
                fb += sum(fv)
                wb += sum(wv)
        if not seen:
            continue
        fb *= scale["FETCH_SIZE"] / steps
        wb *= scale["WRITE_SIZE"] / steps
        table[f"{call}:{workload}"] = {
            "source_sha": source_sha(call), "kernels": seen, "steps": steps,
            "fetch_bytes_per_launch": round(fb), "write_bytes_per_launch": round(wb),
            "hbm_bytes_per_launch": round(fb + wb),
            "fetch_scale": round(scale["FETCH_SIZE"], 4), "write_scale": round(scale["WRITE_SIZE"], 4)}
    with open(p, "w") as f:
        json.dump(table, f, indent=1, sort_keys=True)
        f.write("\n")
    return table


def cpu_sample(w, batch):
    """A bounded sample of batch 0 for the CPU baselines: the first whole
    tables (or, for one table, the first bags) holding about 84M gathered
    floats (a 1.3M-pair batch of 64-float rows, about half a second of
    single-threaded oracle work)."""
    import numpy as np

    from paper_2010_13100_amd import workload as wl
    target_pairs = max(1, 84_000_000 // w.dim)
    bo = batch.bag_offsets
    if batch.num_pairs <= target_pairs:
        tables, bags = w.num_tables, w.batch
    elif w.num_tables > 1:
        per_table = bo[np.arange(1, w.num_tables + 1) * w.batch] - bo[np.arange(w.num_tables)
                                                                      * w.batch]
        tables = max(1, int(np.searchsorted(np.cumsum(per_table), target_pairs, side="right")))
        bags = w.batch
    else:
        tables, bags = 1, max(1, int(np.searchsorted(bo, target_pairs, side="right")) - 1)
    nb = tables * bags
    s_bo = bo[:nb + 1].copy()
    n = int(s_bo[-1])
    s_idx = batch.indices[:n]
    s_off = batch.table_row_offset[:tables + 1].copy()
    t = np.repeat(np.arange(nb) // bags, np.diff(s_bo))
    src = s_off[t] + s_idx
    ids = np.unique(src)
    return dict(tables=tables, bags=bags, bo=s_bo, idx=s_idx, off=s_off, grad=batch.grad_out[:nb],
                n=n, ids=ids, pair_row=np.searchsorted(ids, src).astype(np.int32),
                table=wl.table_rows(w, ids),
                text=f"the first {tables} table(s) x {bags} bags of batch 0: {n} of "
                     f"{batch.num_pairs} pairs, {len(ids)} table rows")


def cpu_baseline(w, batch, budget_s: float, sample=None):
    """The fp32 oracle (single thread) on a bounded sample of the workload
    (cpu_sample): forward, casting, the baseline expand + coalesce backward
    and the update, on the rows the sample touches; steps/s is scaled to the
    full batch by the sample's share of the pairs."""
    import numpy as np

    import oracle
    orc = oracle.Oracle("f32")
    s = sample or cpu_sample(w, batch)
    steps, t0 = 0, time.perf_counter()
    phases: dict = {}
    while True:
        oracle.train_step(orc, num_tables=s["tables"], bags_per_table=s["bags"],
                          table_row_offset=s["off"], indices=s["idx"], bag_offsets=s["bo"],
                          grad_out=s["grad"], table=s["table"], table_ids=s["ids"],
                          optimizer=w.optimizer, lr=np.float32(w.lr), eps=np.float32(w.eps),
                          gamma=np.float32(w.gamma), timings=phases)
        steps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or steps >= 50:
            break
    share = s["n"] / batch.num_pairs
    return {"value": steps / el * share, "unit": "steps/s", "cores": 1, "kind": "oracle",
            "sample": f"{steps} oracle steps (fp32, one thread) on {s['text']}; steps/s "
                      "scaled by that share of the pairs",
            "sample_steps_per_s": round(steps / el, 4),
            "seconds_per_phase": {k: round(v / steps, 4) for k, v in phases.items()}}


def cpu_baseline_allcores(w, batch, budget_s: float, sample=None):
    """The paper's baseline step (forward, expand, stable argsort,
    Algorithm 1, update) on all host cores with OpenMP (cpu_baseline/, equal
    to the oracle bit for bit), on the same sample as cpu_baseline."""
    import numpy as np

    import cpu_baseline as cb_mod
    if w.optimizer not in ("sgd", "adagrad"):
        return None
    cb = cb_mod.CpuBaseline()
    s = sample or cpu_sample(w, batch)
    steps, t0 = 0, time.perf_counter()
    phases: dict = {}
    while True:
        table = s["table"].copy()
        acc = np.zeros_like(table) if w.optimizer == "adagrad" else None
        t1 = time.perf_counter()
        _, _, _, ph = cb.train_step(s["bo"], s["pair_row"], table, s["grad"], w.optimizer, acc,
                                    np.float32(w.lr), np.float32(w.eps))
        for k, v in ph.items():
            phases[k] = phases.get(k, 0.0) + v
        steps += 1
        phases["_step"] = phases.get("_step", 0.0) + time.perf_counter() - t1
        if time.perf_counter() - t0 >= budget_s or steps >= 200:
            break
    step_s = phases.pop("_step") / steps
    share = s["n"] / batch.num_pairs
    return {"value": 1.0 / step_s * share, "unit": "steps/s", "cores": cb.threads,
            "kind": "openmp expand-coalesce (the paper's baseline step, all host cores)",
            "sample": f"{steps} steps on {s['text']} (table copy per step not timed); "
                      "steps/s scaled by that share of the pairs",
            "sample_steps_per_s": round(1.0 / step_s, 4),
            "seconds_per_phase": {k: round(v / steps, 5) for k, v in phases.items()}}


def setup(w, dev):
    """Batches, a trainer with a filled table, and device copies of the
    batches for workload w."""
    import torch

    from paper_2010_13100_amd import device_fill, tc
    from paper_2010_13100_amd import workload as wl

    print(f"[bench] workload {w.name}: generating {NUM_BATCHES} batches", file=sys.stderr,
          flush=True)
    batches = [wl.make_batch(w, step=s) for s in range(NUM_BATCHES)]
    max_pairs = max(b.num_pairs for b in batches)
    trainer = tc.EmbeddingTrainer(total_rows=w.total_rows, dim=w.dim, num_tables=w.num_tables,
                                  bags_per_table=w.batch, max_pairs=max_pairs,
                                  optimizer=w.optimizer, lr=w.lr, eps=w.eps, gamma=w.gamma,
                                  device=dev, max_table_rows=w.rows_per_table)
    device_fill.fill_uniform(trainer.W, seed=0, lo=w.init_lo, hi=w.init_hi)
    dbat = [dict(off=torch.from_numpy(b.table_row_offset).to(dev),
                 idx=torch.from_numpy(b.indices).to(dev),
                 bo=torch.from_numpy(b.bag_offsets).to(dev),
                 grad=torch.from_numpy(b.grad_out).to(dev), n=b.num_pairs) for b in batches]
    return batches, trainer, dbat


def measure_step(args, w, cfg_name, trainer, dbat, stream, calls, traffic_key):
    """Time args.steps steps (after args.warmup) of the given calls and
    return the result line (without cpu_baseline)."""
    import numpy as np
    import torch

    fns = {"forward": lambda d: trainer.forward(d["off"], d["idx"], d["bo"], stream),
           "cast": lambda d: trainer.cast(d["off"], d["idx"], d["bo"], d["n"], stream),
           "forward_cast": lambda d: trainer.forward_cast(d["off"], d["idx"], d["bo"], d["n"],
                                                          stream),
           "backward": lambda d: trainer.backward(d["grad"], stream),
           "update": lambda d: trainer.update(stream),
           "backward_update": lambda d: trainer.backward_update(d["grad"], stream)}

    def step(i, ev=None):
        """One step on batch i % NUM_BATCHES. ev: dict call -> (start, stop)
        events to record around that call (each record is a marker on the
        stream, so the timed steps record only the dominant call's pair)."""
        d = dbat[i % NUM_BATCHES]
        for c in calls:
            e = ev.get(c) if ev else None
            if e:
                e[0].record(stream)
            fns[c](d)
            if e:
                e[1].record(stream)

    def ev_pair():
        return (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))

    if args.profile_steps:
        # for profiler runs: the step calls only, nothing else on the GPU
        for i in range(args.warmup + args.steps):
            step(i)
        torch.cuda.synchronize()
        return None

    # warm-up steps, every call timed: per-call durations and the dominant call
    print(f"[bench] {cfg_name}: warmup {args.warmup} steps", file=sys.stderr, flush=True)
    wev = [{c: ev_pair() for c in calls} for _ in range(args.warmup)]
    for i in range(args.warmup):
        step(i, wev[i])
    torch.cuda.synchronize()
    skip = 1 if args.warmup > 1 else 0   # the first step also pays one-time costs
    per_call_ms = {c: float(np.mean([e[c][0].elapsed_time(e[c][1]) for e in wev[skip:]]))
                   for c in calls} if args.warmup else {c: float("nan") for c in calls}
    # the dominant call: the longest one of the step
    dom = max(calls, key=lambda c: per_call_ms[c]) if args.warmup else calls[-1]

    # timed steps: start/stop around the whole region, one event pair around
    # the dominant call of each step (on the stream its kernels run on)
    tev = [{dom: ev_pair()} for _ in range(args.steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for i in range(args.steps):
        step(args.warmup + i, tev[i])
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_total = start.elapsed_time(stop)
    ms_step = ms_total / args.steps
    dom_ms = float(np.mean([e[dom][0].elapsed_time(e[dom][1]) for e in tev]))
    print(f"[bench] {cfg_name}: timed {args.steps} steps: {ms_step:.4f} ms/step "
          f"(wall {wall:.3f} s)", file=sys.stderr, flush=True)

    # unique rows and longest segment per batch (outside the timed region)
    uniq, longest = [], []
    for i in range(NUM_BATCHES):
        d = dbat[i]
        trainer.cast(d["off"], d["idx"], d["bo"], d["n"], stream)
        u = int(trainer.num_unique.item())
        so = trainer.seg_offsets[:u + 1]
        uniq.append(u)
        longest.append(int((so[1:] - so[:-1]).max().item()) if u else 0)
    alg = {c: 0.0 for c in calls}
    comp = {c: 0.0 for c in calls}
    for i in range(args.steps):
        b = (args.warmup + i) % NUM_BATCHES
        a = algorithmic_bytes(w, dbat[b]["n"], uniq[b], w.num_bags)
        m = compulsory_bytes(w, dbat[b]["n"], uniq[b], w.num_bags)
        for c in calls:
            alg[c] += a[c] / args.steps
            comp[c] += m[c] / args.steps
    step_alg, step_comp = sum(alg.values()), sum(comp.values())
    step_s = ms_step * 1e-3

    counted = {c: None if traffic_key is None else load_traffic(c, traffic_key) for c in calls}
    step_counted = (None if any(v is None for v in counted.values())
                    else float(sum(counted.values())))
    achieved = alg[dom] / (dom_ms * 1e-3) / 1e9
    traffic = counted[dom]
    traffic_gbs = None if traffic is None else traffic / (dom_ms * 1e-3) / 1e9

    def frac(nbytes, sec):
        return None if nbytes is None else round(nbytes / sec / 1e9 / HBM_PEAK_GBS, 4)

    call_name = {"update": "tc_sparse_update", "cast": "tc_cast_index"}
    return {
        "metric": "embedding train steps/sec (fwd+cast+bwd+update) and achieved HBM GB/s",
        "value": round(args.steps / (ms_total * 1e-3), 3),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded Zipf/uniform index streams, N(0,1) output gradients, "
                "SplitMix64 table init)",
        "config": {"workload": f"{cfg_name}: {w.name}", "tables": w.num_tables,
                   "rows_per_table": w.rows_per_table, "dim": w.dim, "batch": w.batch,
                   "pairs_per_step": round(float(np.mean([d["n"] for d in dbat])), 1),
                   "unique_rows_per_step": round(float(np.mean(uniq)), 1),
                   "longest_segment": max(longest),
                   "optimizer": w.optimizer,
                   "step_calls": calls},
        # the whole step against the HBM peak, three ways: the paper's traffic
        # model (every gather counted), the byte counters (rocprofv3
        # FETCH_SIZE + WRITE_SIZE, scaled), and the compulsory bound (every
        # distinct row once)
        "step_hbm": {
            "algorithmic_bytes": round(step_alg),
            "algorithmic_frac": frac(step_alg, step_s),
            "counter_bytes": None if step_counted is None else round(step_counted),
            "counter_frac": frac(step_counted, step_s),
            "compulsory_bytes": round(step_comp),
            "compulsory_frac": frac(step_comp, step_s),
            "peak_GBps": HBM_PEAK_GBS},
        "per_call_us": {c: round(v * 1e3, 2) for c, v in per_call_ms.items()},
        "per_call_us_measured_on": f"warm-up steps {skip}..{args.warmup - 1}, every call timed",
        "per_call_algorithmic_GBps": {c: round(alg[c] / (per_call_ms[c] * 1e-3) / 1e9, 1)
                                      for c in calls},
        "per_call_counter_GBps": {c: None if counted[c] is None
                                  else round(counted[c] / (per_call_ms[c] * 1e-3) / 1e9, 1)
                                  for c in calls},
        "roofline": {"bound": "hbm", "call": call_name.get(dom, f"tc_embed_{dom}"),
                     "kernels": KERNEL_NAMES[dom],
                     "launch_us": round(dom_ms * 1e3, 2),
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic,
                     "traffic_GBps": None if traffic_gbs is None else round(traffic_gbs, 1),
                     "traffic_frac": None if traffic_gbs is None
                     else round(traffic_gbs / HBM_PEAK_GBS, 4),
                     "compulsory_frac": frac(comp[dom], dom_ms * 1e-3)},
    }


def compact(res):
    """The fields of a side workload's result kept in the headline line."""
    r = res["roofline"]
    return {"workload": res["config"]["workload"], "steps_per_s": res["value"],
            "ms_per_step": res["ms_per_step"], "per_call_us": res["per_call_us"],
            "pairs_per_step": res["config"]["pairs_per_step"],
            "unique_rows_per_step": res["config"]["unique_rows_per_step"],
            "longest_segment": res["config"]["longest_segment"],
            "step_hbm": {k: v for k, v in res["step_hbm"].items() if k.endswith("frac")},
            "dominant_call": r["call"], "dominant_algorithmic_frac": r["frac"],
            "dominant_counter_frac": r["traffic_frac"],
            "dominant_compulsory_frac": r["compulsory_frac"],
            **({"pipelined": res["pipelined"]} if "pipelined" in res else {})}


def run_sweep(args, base, cfg_name, dev):
    """The sensitivity study (Sec. VI-D): for each batch size or embedding
    dimension, the step (steps/s, dominant call's HBM fraction) and the
    backward A/B (baseline expand-coalesce against Tensor Casting). One JSON
    line per point."""
    import torch

    from paper_2010_13100_amd import workload as wl

    what, _, values = args.sweep.partition("=")
    if what not in ("batch", "dim") or not values:
        raise SystemExit("--sweep takes batch=B1,B2,... or dim=D1,D2,...")
    for v in (int(x) for x in values.split(",")):
        w = wl.variant(base, **{what: v})
        _, trainer, dbat = setup(w, dev)
        stream = torch.cuda.current_stream(dev)
        res = measure_step(args, w, cfg_name, trainer, dbat, stream, step_calls(args, w), None)
        ab = run_ab(args, w, trainer, dbat, stream)
        print(json.dumps({
            "sweep": what, what: v, "workload": w.name,
            "pairs_per_step": res["config"]["pairs_per_step"],
            "unique_rows_per_step": res["config"]["unique_rows_per_step"],
            "steps_per_s": res["value"], "ms_per_step": res["ms_per_step"],
            "per_call_us": res["per_call_us"],
            "dominant_call": res["roofline"]["call"],
            "dominant_frac_of_hbm_peak": res["roofline"]["frac"],
            "step_hbm": res["step_hbm"],
            "ab_baseline_us": ab["baseline_us"], "ab_casted_us": ab["casted_us"],
            "ab_speedup": ab["speedup"], "ab_bytes_ratio": ab["algorithmic_bytes"]["ratio"],
            "steps": args.steps, "warmup": args.warmup}), flush=True)
        del trainer, dbat
        torch.cuda.synchronize()
        torch.cuda.empty_cache()


def measure_pipelined(args, trainer, dbat, stream, mode):
    """Steps with the next batch's cast on a side stream (the paper's
    decoupled casting, Sec. IV-B, across steps), into a second slot of cast
    outputs; the forward runs as its own call. mode "step": cast(i + 1)
    beside forward(i) and backward + update(i) (it waits only for the
    backward of step i - 1, the last reader of its slot); mode "backward":
    cast(i + 1) waits for forward(i) and runs beside backward + update(i).
    Same table bits as the stream-ordered step. Returns steps/s and ms/step
    over args.steps steps (after args.warmup)."""
    import torch

    side = torch.cuda.Stream()
    trainer.cast_slots(2)

    def run(i0, n):
        e_cast = [torch.cuda.Event() for _ in range(n)]
        e_mark = [torch.cuda.Event() for _ in range(n)]
        d0 = dbat[i0 % NUM_BATCHES]
        trainer.cast(d0["off"], d0["idx"], d0["bo"], d0["n"], stream, slot=i0 % 2)
        e_cast[0].record(stream)
        for k in range(n):
            i = i0 + k
            d = dbat[i % NUM_BATCHES]
            if mode == "backward":
                stream.wait_event(e_cast[k])
                trainer.forward(d["off"], d["idx"], d["bo"], stream)
                e_mark[k].record(stream)
            if k + 1 < n:
                dn = dbat[(i + 1) % NUM_BATCHES]
                with torch.cuda.stream(side):
                    if mode == "backward":
                        side.wait_event(e_mark[k])
                    else:
                        side.wait_event(e_mark[k - 1] if k >= 1 else e_cast[0])
                    trainer.cast(dn["off"], dn["idx"], dn["bo"], dn["n"], side,
                                 slot=(i + 1) % 2)
                    e_cast[k + 1].record(side)
            if mode == "step":
                stream.wait_event(e_cast[k])
                trainer.forward(d["off"], d["idx"], d["bo"], stream)
            trainer.backward_update(d["grad"], stream, slot=i % 2)
            if mode == "step":
                e_mark[k].record(stream)

    if args.warmup:
        run(0, args.warmup)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    run(args.warmup, args.steps)
    stop.record(stream)
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(stop) / args.steps
    return {"schedule": mode, "steps_per_s": round(1000.0 / ms_step, 3),
            "ms_per_step": round(ms_step, 5)}


def run_workload(args, cfg_name, dev, keep_batch=False):
    """Set up one workload, time its step, free its device memory. Returns
    (result line, batch 0 if keep_batch else None)."""
    import torch

    from paper_2010_13100_amd import workload as wl

    w = wl.WORKLOADS[cfg_name]
    variant = wl.variant(w, batch=args.batch, dim=args.dim, optimizer=args.optimizer)
    traffic_key = cfg_name if variant is w and not args.no_overlap and not args.unfused else None
    w = variant
    batches, trainer, dbat = setup(w, dev)
    stream = torch.cuda.current_stream(dev)
    res = measure_step(args, w, cfg_name, trainer, dbat, stream, step_calls(args, w),
                       traffic_key)
    if args.pipeline != "none" and w.optimizer != "rowwise_adagrad":
        print(f"[bench] {cfg_name}: pipelined cast ({args.pipeline})", file=sys.stderr,
              flush=True)
        res["pipelined"] = measure_pipelined(args, trainer, dbat, stream, args.pipeline)
    keep = batches[0] if keep_batch else None
    del trainer, dbat, batches
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res, keep, w


def run_forward_span(args, w, dev, spans):
    """The forward gather-reduce alone on the workload's shape with each
    table's row ids drawn uniformly from its first R rows, for each R in
    spans: how the gather rate depends on the address range the random
    row reads cover (translation reach, caches). One JSON line per span."""
    import numpy as np
    import torch

    from paper_2010_13100_amd import device_fill, tc

    T, B, D = w.num_tables, w.batch, w.dim
    W = torch.empty((w.total_rows, D), dtype=torch.float32, device=dev)
    device_fill.fill_uniform(W, seed=0, lo=w.init_lo, hi=w.init_hi)
    lengths = np.full(T * B, w.pooling_value, np.int64)
    bo = torch.from_numpy(np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)).to(dev)
    off = torch.from_numpy(np.arange(T + 1, dtype=np.int64) * w.rows_per_table).to(dev)
    out = torch.empty((T * B, D), dtype=torch.float32, device=dev)
    rng = np.random.default_rng(0)
    n = int(lengths.sum())
    for span in spans:
        span = min(span, w.rows_per_table)
        idx = torch.from_numpy(rng.integers(0, span, size=n).astype(np.int32)).to(dev)
        for _ in range(args.warmup):
            tc.tc_embed_forward(W, off, T, B, idx, bo, out)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            tc.tc_embed_forward(W, off, T, B, idx, bo, out)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / args.steps
        nbytes = n * (4 + 4 * D) + (T * B + 1) * 4 + T * B * 4 * D
        print(json.dumps({"forward_span_rows": span, "span_MB_per_table": span * D * 4 / 1e6,
                          "workload": w.name, "us": round(us, 1),
                          "algorithmic_GBps": round(nbytes / us / 1e3, 1),
                          "frac_of_hbm_peak": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4)}),
              flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="c4", choices=["c1", "c2", "c3", "c4", "c5"],
                    help="the headline workload (default c4, the largest on one GPU)")
    ap.add_argument("--also", default="c3,c5,c2,c1",
                    help="workloads timed after the headline one, reported compactly in "
                         "the same line under other_workloads ('' for none)")
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of oracle work for cpu_baseline (0 disables)")
    ap.add_argument("--ab", action="store_true",
                    help="instead of the step: time the paper's baseline backward "
                         "(expand-coalesce) against the casted backward and exit")
    ap.add_argument("--unfused", action="store_true",
                    help="every step a call of its own: tc_embed_forward, tc_cast_index, "
                         "tc_embed_backward, tc_sparse_update")
    ap.add_argument("--no-overlap", action="store_true",
                    help="forward and cast as two calls (tc_embed_forward, tc_cast_index)")
    ap.add_argument("--pipeline", default="backward", choices=["step", "backward", "none"],
                    help="also time steps with the next batch's cast on a side stream, beside "
                         "its backward + update ('backward', the default) or beside the whole "
                         "step ('step'); reported under 'pipelined' beside the stream-ordered "
                         "step, which stays the line's value ('none' skips it)")
    ap.add_argument("--optimizer", default=None,
                    choices=["sgd", "adagrad", "rmsprop", "rowwise_adagrad"],
                    help="replace the workload's optimizer (row-wise Adagrad runs unfused)")
    ap.add_argument("--batch", type=int, default=None,
                    help="replace the workload's bags per table")
    ap.add_argument("--dim", type=int, default=None,
                    help="replace the workload's embedding dimension")
    ap.add_argument("--sweep", default=None, metavar="batch=B1,B2,..|dim=D1,D2,..",
                    help="sensitivity sweep: step and backward A/B per value, one JSON line "
                         "each, then exit")
    ap.add_argument("--forward-span", default=None, metavar="R1,R2,..",
                    help="time the forward alone on --config's shape with each table's rows "
                         "drawn from its first R rows, per R, one JSON line each, then exit")
    ap.add_argument("--profile-steps", action="store_true",
                    help="for profiler runs: run warmup + steps steps of --config and "
                         "nothing else on the GPU (no events, no extra casts), print one "
                         "line and exit")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run 5 plain device copies of BYTES bytes (scale for the HBM "
                         "byte counters) and exit")
    ap.add_argument("--traffic-from", metavar="PMC_DIR", default=None,
                    help="write profiles/traffic.json entries for --config from rocprofv3 "
                         "counter runs in PMC_DIR and exit (no GPU needed)")
    args = ap.parse_args()
    if args.traffic_from:
        print(json.dumps(write_traffic(args.traffic_from, args.config,
                                       ["forward_cast", "backward_update"]), indent=1))
        return
    if args.copy_calibration:
        import torch
        src = torch.ones(args.copy_calibration // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": args.copy_calibration, "copies": 5}))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the hot path is built and timed on a single "
              "MI355X; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2010_13100_amd import workload as wl

    dev = torch.device("cuda", 0)
    if args.forward_span:
        run_forward_span(args, wl.WORKLOADS[args.config], dev,
                         [int(x) for x in args.forward_span.split(",")])
        return
    if args.sweep or args.ab or args.profile_steps:
        w = wl.variant(wl.WORKLOADS[args.config], batch=args.batch, dim=args.dim,
                       optimizer=args.optimizer)
        if args.sweep:
            run_sweep(args, w, args.config, dev)
            return
        _, trainer, dbat = setup(w, dev)
        stream = torch.cuda.current_stream(dev)
        if args.ab:
            print(json.dumps(run_ab(args, w, trainer, dbat, stream)), flush=True)
        else:
            measure_step(args, w, args.config, trainer, dbat, stream, step_calls(args, w), None)
            print(json.dumps({"profile_steps": args.warmup + args.steps,
                              "workload": args.config, "calls": step_calls(args, w)}),
                  flush=True)
        return

    result, batch0, w = run_workload(args, args.config, dev, keep_batch=args.cpu_budget > 0)
    others = [c for c in args.also.split(",") if c and c != args.config]
    result["other_workloads"] = {}
    for c in others:
        res, _, _ = run_workload(args, c, dev)
        result["other_workloads"][c] = compact(res)
    result["host"] = host_cpu()
    if args.cpu_budget > 0:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        sample = cpu_sample(w, batch0)
        result["cpu_baseline"] = cpu_baseline(w, batch0, args.cpu_budget, sample)
        print("[bench] timing the all-cores CPU baseline", file=sys.stderr, flush=True)
        result["cpu_baseline_allcores"] = cpu_baseline_allcores(w, batch0, args.cpu_budget / 2,
                                                                sample)
    else:
        result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
