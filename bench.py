#!/usr/bin/env python3
"""Throughput of the belief-update hot path on one MI355X.

Workload: the large shared-model case -- F = 4 hidden factors of 32 states
(4 actions each), M = 4 modalities of 32 outcomes that each depend on all four
factors (32^5 entries per A_m, 90% random zeros, renormalised columns), one
model shared by b = 64 agents, window T = 16, 16 iterations.  One step runs
VMP and MMP over the whole batch on both A layouts:
  dense  (BI_DENSE_A | BI_FAST_F32 | BI_F16_PAIRS): the slices stored as fp16
         (high, residual) pairs, contracted on fp16 matrix cores with three
         products per fp32 product and fp32 accumulation; fp64 message sums /
         transitions / softmax (--dense-f32: fp32 matrix cores on the fp32
         copy instead);
  sparse (BI_SPARSE_A | BI_FAST_F32 | BI_F16_PAIRS): the nonzeros stored as
         fp16 pairs (8 bytes each) in blocks of 64 lines, scattered per
         first-factor state into LDS and contracted on the same fp16 matrix
         cores (--sparse-f64: fp64 gathers over the nonzero entries instead).
The two layouts' calls share nothing but the GPU, so a step runs each
layout's calls (VMP, then MMP) on a stream of its own, forked from and joined
back to the timing stream: the HBM-bound dense calls overlap the
instruction-bound sparse ones.  The record also carries the same step with
every call on one stream (`serial`); the per-kernel and per-call passes run
serially.  Inputs are resident in HBM before timing starts; each model is
packed once outside the timed region (the one-time layout step).  After the
set-up the step runs 30 untimed settle steps, then the --warmup steps, then
the timed --steps.

Prints one JSON line.  value = belief updates per second over the whole job,
one belief update being one (agent, time step, iteration) of one algorithm
on one layout.

--workload picks another workload for measurement (agent-resident fp64
kernels, one model per agent): vmp_2f (F=2 factors of 8 and 6 states, M=3
modalities on both, T=10, b=1024, VMP), mmp_3f (F=3 of 12/10/8 states, M=4 x
16 outcomes on random factor subsets, T=20, b=4096, MMP), fpi_hmm (one
4-state factor, T=8, b=1, FPI), fpi_2f (FPI on the F=2 models), fpi_2f_rolling
(the same, online: T calls of one step, each carrying the predictive prior of
the step before through bi_predict), mmp_3f_bdeps (the F=3 structure with
every factor's transition conditioned on itself and one other factor).  --soft
runs a workload (the large one too) with soft observation vectors (each puts
0.7 on the sampled outcome and spreads the rest as a Dirichlet(1) draw)
through bi_infer_soft.
"""
import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "belief updates/sec (agents×timesteps×iters) + achieved HBM GB/s, 1 MI355X"
PEAK_FP32_MFMA_TFLOPS = 157.3
PEAK_FP16_MFMA_TFLOPS = 2500.0
PEAK_FP64_VALU_TFLOPS = 78.6
PEAK_HBM_GBPS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_large_shared.json")
CSRC = os.path.join(ROOT, "paper_2607_17855_amd", "csrc")
# likelihood kernels: profile class -> (kernel symbol, source file)
LIK = {"lik": ("lik_kernel", "stream.hip"), "lik_split": ("split_lik_kernel<false>", "split.hip"),
       "lik_split16": ("split_lik_kernel<true>", "split.hip"), "lik_sparse": ("sparse_lik_kernel", "sparse.hip"),
       "lik_sparse16": ("sparse16_lik_kernel", "split.hip"),
       "lik_rowcol16": ("rowcol16_lik_kernel", "rowcol.hip")}
LAYOUTS = ("dense", "sparse")
ALGOS = ("vmp", "mmp")


def source_sha(fname: str) -> str:
    with open(os.path.join(CSRC, fname), "rb") as fh:
        return hashlib.sha256(fh.read()).hexdigest()[:16]


import numpy as np   # noqa: E402  (host-side arithmetic of the work counts)


def slice_sizes(model):
    out = []
    for d in model.deps:
        P = 1
        for f in d:
            P *= model.n[f]
        out.append(P)
    return out


def outcome_counts(model, obs, soft=None):
    """Per modality, how many contexts apply each outcome's slice in a
    likelihood launch: the contexts observing it, or with soft vectors
    [b][T][sum K] the contexts whose vector weights it (nonzero)."""
    import numpy as np
    if soft is None:
        return [np.bincount(obs[:, :, m].ravel(), minlength=model.K[m]) for m in range(model.M)]
    offs = np.cumsum([0] + list(model.K))
    return [(soft[:, :, offs[m]:offs[m + 1]] != 0).reshape(-1, model.K[m]).sum(axis=0) for m in range(model.M)]


def dense_lik_work(model, obs, soft=None):
    """Algorithmic flops and HBM bytes of one dense likelihood launch: per
    context (soft vectors: per weighted outcome of a context) and modality the
    two contractions of the slice (towards its rows and towards its columns),
    one FMA (2 flops) per slice entry each (16.8 MFLOP per belief update with
    outcomes); every slice applied by at least one context is read once in
    fp32."""
    import numpy as np
    cnts = outcome_counts(model, obs, soft)
    P = slice_sizes(model)
    flops = sum(2 * 2 * p * float(c.sum()) for p, c in zip(P, cnts))
    nbytes = sum(4.0 * p * int((c > 0).sum()) for p, c in zip(P, cnts))
    return float(flops), float(nbytes)


def sparse_lik_work(model, obs, soft=None):
    """Algorithmic flops and HBM bytes of one sparse likelihood launch: for
    every context, each nonzero of its observed slices is visited twice (row
    lines and column lines), one multiply and one FMA (3 flops) each; every
    observed slice's entries are read once per side (16 B per entry and side)."""
    import numpy as np
    flops = 0.0
    nbytes = 0.0
    for m, cnt in enumerate(outcome_counts(model, obs, soft)):
        A = model.A[m][0].reshape(model.K[m], -1)
        nnz = (A.astype(np.float64) > 1e-16).sum(axis=1)
        flops += 2 * 3 * float((nnz * cnt).sum())
        nbytes += 2 * 16.0 * float(nnz[cnt > 0].sum())
    return flops, nbytes


def sparse16_lik_work(model, obs, soft=None):
    """Algorithmic flops and HBM bytes of one sparse fp16-pair likelihood
    launch: the flops of the dense contractions (the matrix cores run the
    zeros too; 3 fp16 products per fp32 product come on top), and every
    observed slice's nonzeros read once, 8 B each (value and position), the
    minimum a sparse layout moves.  The layout stores each nonzero once per
    side (rows and columns) and the kernel reads both copies: that figure is
    returned third."""
    import numpy as np
    flops, _ = dense_lik_work(model, obs, soft)
    nbytes = 0.0
    for m, cnt in enumerate(outcome_counts(model, obs, soft)):
        A = model.A[m][0].reshape(model.K[m], -1)
        nnz = (A.astype(np.float64) > 1e-16).sum(axis=1)
        nbytes += 8.0 * float(nnz[cnt > 0].sum())
    return flops, nbytes, 2 * nbytes


def agent_work(model, T, algo):
    """Algorithmic flops and bytes of one belief update on the agent-resident
    path: the two contractions of every observed slice (one FMA per entry
    each), the transition messages (per state of f: the forward contraction
    over the states of f's B-dependency list, and for every factor j whose
    list holds f the backward one over s_{t+1}^j and j's other listed
    factors; two n x n products per factor for trivial lists; FPI: the
    forward one only, once per time step, counted per update), and one read
    of the observed fp64 slices."""
    lik = sum(4 * P for P in slice_sizes(model))
    bstates = [int(np.prod([model.n[g] for g in model.bdep(f)])) for f in range(model.F)]
    trans = 0
    for f, n in enumerate(model.n):
        fwd = n * bstates[f]
        bwd = sum(model.n[j] * bstates[j] for j in range(model.F) if f in model.bdep(j))   # n states x n_j x others
        trans += 2 * (fwd if algo == "fpi" else fwd + bwd)
    nbytes = sum(8.0 * P for P in slice_sizes(model))
    return float(lik + trans), nbytes


# per-agent workloads: name -> (generator, algorithm, options)
# untimed steps run after set-up and before the --warmup steps (large workload)
SETTLE_STEPS = 30

AGENT_WORKLOADS = {
    "vmp_2f": ("two_factor_agents", "vmp", {}),
    "mmp_3f": ("three_factor_agents", "mmp", {}),
    "fpi_hmm": ("hmm_small", "fpi", {}),
    # the F=2 models filtered over the whole window, and online: one step per
    # call, each carrying the predictive prior of the step before (bi_predict)
    "fpi_2f": ("two_factor_agents", "fpi", {}),
    "fpi_2f_rolling": ("two_factor_agents", "fpi", {"rolling": True}),
    # the F=3 structure with coupled transitions (B-dependency lists)
    "mmp_3f_bdeps": ("three_factor_agents", "mmp", {"bdeps": True}),
}


def soft_ll_bytes(model, b, T):
    """Algorithmic HBM bytes of one soft log-likelihood launch: the fp64
    slices of every outcome read once per agent (once in all for a shared
    model) and T expected log-likelihood tensors written per agent."""
    P = slice_sizes(model)
    reads = sum(8.0 * k * p for k, p in zip(model.K, P)) * (1 if model.mb == 1 else b)
    return reads + 8.0 * b * T * sum(P)


def cpu_baseline(w, algos, budget_s: float = 25.0, soft=None, keep: bool = False, min_s: float = 1.0):
    """The oracle timed on the host cores over a bounded sample of agents (a
    sample shorter than min_s is repeated, its first pass untimed, so a tiny
    workload is not timed on its first-call overhead).
    keep: also return its outputs {algo: q [agents][T][sum n]} and the agents."""
    import numpy as np
    import oracle
    threads = oracle.default_threads()
    n_agents = max(1, min(w.b, threads))
    agents = list(np.linspace(0, w.b - 1, n_agents).astype(int))

    def run(algo, ags):
        if soft is None:
            return oracle.infer(algo, w.model, w.obs, w.act, w.iters, agents=ags)
        return oracle.infer_soft(algo, w.model, soft, w.act, w.iters, agents=ags)

    outs = {}

    def sample():
        t0 = time.perf_counter()
        done, calls = 0, 0
        for algo in algos:
            outs[algo] = run(algo, agents)
            done += len(agents) * w.T * w.iters
            calls += 1
            if time.perf_counter() - t0 > budget_s:
                break
        return done, calls, time.perf_counter() - t0

    done_bu, calls, dt = sample()
    passes = 1
    if dt < min_s and calls == len(algos):
        # short: that pass was the warm-up; repeat the timed passes
        t0 = time.perf_counter()
        done_bu, passes = 0, 0
        while time.perf_counter() - t0 < min_s:
            done_bu += sample()[0]
            passes += 1
        dt = time.perf_counter() - t0
    res = {"value": done_bu / dt, "unit": "belief_updates/s", "cores": min(threads, len(agents)),
           "kind": "oracle",
           "sample": f"{len(agents)} of {w.b} agents x T={w.T} x {w.iters} iters, "
                     f"{'+'.join(algos[:calls])}{' (soft observations)' if soft is not None else ''}"
                     f"{f' x {passes} passes' if passes > 1 else ''}, "
                     f"fp64 looped oracle (layout-independent), {dt:.1f} s wall"}
    return (res, outs, agents) if keep else res


def cpu_baseline_1thread(w, algo, min_s: float = 1.0):
    """The oracle on one host thread, one agent (a call shorter than min_s is
    repeated, the first one untimed)."""
    import oracle
    t0 = time.perf_counter()
    oracle.infer(algo, w.model, w.obs, w.act, w.iters, agents=[0], threads=1)
    dt = time.perf_counter() - t0
    reps = 1
    if dt < min_s:
        t0 = time.perf_counter()
        reps = 0
        while time.perf_counter() - t0 < min_s:
            oracle.infer(algo, w.model, w.obs, w.act, w.iters, agents=[0], threads=1)
            reps += 1
        dt = time.perf_counter() - t0
    return {"value": reps * w.T * w.iters / dt, "unit": "belief_updates/s", "cores": 1, "kind": "oracle",
            "sample": f"agent 0 x T={w.T} x {w.iters} iters x {reps}, {algo}, {dt:.1f} s wall"}


def load_agent_traffic():
    path = os.path.join(ROOT, "profiles", "traffic_agent.json")
    if not os.path.exists(path):
        return {}
    with open(path) as fh:
        return json.load(fh)


def load_traffic():
    if not os.path.exists(TRAFFIC_FILE):
        return {}
    with open(TRAFFIC_FILE) as fh:
        return json.load(fh)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--layouts", default=",".join(LAYOUTS), help="comma list of A layouts in a step")
    ap.add_argument("--workload", default="large", choices=["large", "sweep"] + list(AGENT_WORKLOADS))
    ap.add_argument("--regimes", default="uniform,skewed", help="sweep workload: dimension regimes")
    ap.add_argument("--cases", default="0:770", help="sweep workload: start:stop of the seeded specs")
    ap.add_argument("--soft", action="store_true",
                    help="soft observation vectors instead of outcomes (every outcome weighted)")
    ap.add_argument("--dense-f32", action="store_true",
                    help="dense layout on fp32 matrix cores (the fp32 copy) instead of the fp16 pairs")
    ap.add_argument("--sparse-f64", action="store_true",
                    help="sparse layout on the fp64 gather kernels instead of the fp16-pair matrix-core tiles")
    ap.add_argument("--serial", action="store_true",
                    help="large workload: every call of a step on one stream (no overlap of the layouts' calls)")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the step on the other precision classes (fp32 matrix cores, fp64 sparse gathers)")
    ap.add_argument("--cache-probe", action="store_true",
                    help="only print copy bandwidth against working-set size (memory-side cache)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="also run a device-to-device copy of MIB MiB (reference kernel for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: runs on one GPU only (agents are independent: a multi-GPU job shards them "
              "across GPUs with no communication)", file=sys.stderr)
        sys.exit(2)
    layouts = [x for x in args.layouts.split(",") if x]
    assert set(layouts) <= set(LAYOUTS) and layouts, f"layouts must be among {LAYOUTS}"

    import torch
    from paper_2607_17855_amd import bi, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.cache_probe:
        return cache_probe(torch, dev)
    if args.workload == "sweep":
        return bench_sweep(args, bi, synth, torch, dev)
    if args.workload != "large":
        return bench_agent(args, bi, synth, torch, dev)
    w = synth.large_shared()
    import numpy as np
    soft_np = (synth.soft_obs(np.random.Generator(np.random.PCG64(17855)), w.obs, w.model.K, confidence=0.7)
               if args.soft else None)
    soft_dev = torch.from_numpy(soft_np).to(dev) if args.soft else None
    fast = {"dense": bi.BI_DENSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS,
            "sparse": bi.BI_SPARSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS}
    plain = {"dense": bi.BI_DENSE_A | bi.BI_FAST_F32, "sparse": bi.BI_SPARSE_A}   # fp32 MFMA / fp64 gathers
    flags = {"dense": plain["dense"] if args.dense_f32 else fast["dense"],
             "sparse": plain["sparse"] if args.sparse_f64 else fast["sparse"]}
    obs = torch.from_numpy(w.obs).to(dev)
    act = torch.from_numpy(w.act).to(dev)
    stream = torch.cuda.current_stream()

    def setup(fl):
        pms = {lay: bi.PackedModel(w.model, flags=fl[lay], device=dev) for lay in layouts}
        qs = {(lay, a): torch.empty((w.b, w.T, w.model.n_total), dtype=torch.float32, device=dev)
              for lay in layouts for a in ALGOS}
        wss = {(lay, a): (pms[lay].workspace_soft if args.soft else pms[lay].workspace)(w.b, w.T, a)
               for lay in layouts for a in ALGOS}
        for key, ws in wss.items():
            assert ws is not None, f"{key}: the large shared model must run on the streaming kernels"
        for a in ALGOS:
            if "sparse" in layouts:
                assert pms["sparse"].path(w.b, w.T, a) == "sparse", "the sparse layout must run the sparse kernels"
        return pms, qs, wss

    # the layouts' calls share nothing but the GPU: the headline step runs
    # each layout's calls (VMP, then MMP) on a stream of its own, forked from
    # and joined back to the timing stream (default priority), so the
    # HBM-bound dense calls and the instruction-bound sparse ones overlap
    side = {lay: torch.cuda.Stream(device=dev) for lay in layouts}

    def make_step(pms, qs, wss):
        def call(lay, a, st):
            if args.soft:
                pms[lay].infer_soft(a, soft_dev, act, w.iters, q=qs[(lay, a)], ws=wss[(lay, a)], stream=st)
            else:
                pms[lay].infer(a, obs, act, w.iters, q=qs[(lay, a)], ws=wss[(lay, a)], stream=st)

        def step(st=stream, marks=None, serial=False):
            if not (serial or args.serial) and marks is None and st is not None and len(layouts) > 1:
                fork = torch.cuda.Event()
                fork.record(st)
                for lay in layouts:
                    side[lay].wait_event(fork)
                    for a in ALGOS:
                        call(lay, a, side[lay])
                for lay in layouts:
                    join = torch.cuda.Event()
                    join.record(side[lay])
                    st.wait_event(join)
                return
            for lay in layouts:
                for a in ALGOS:
                    if marks is not None:
                        marks[(lay, a)][0].record(st)
                    call(lay, a, st)
                    if marks is not None:
                        marks[(lay, a)][1].record(st)
        return step

    def timed(step, serial=False):
        """ms per step over args.steps steps, nothing else on the streams."""
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ev0.record(stream)
        for _ in range(args.steps):
            step(serial=serial)
        ev1.record(stream)
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) / args.steps, time.perf_counter() - t0

    if args.copy_calibration > 0:
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    pms, qs, wss = setup(flags)
    step = make_step(pms, qs, wss)
    # untimed settle steps after the set-up (the first ~100 ms of steps after
    # packing showed occasional host stalls of 20-30 ms), then the warm-up
    for _ in range(SETTLE_STEPS + args.warmup):
        step()
    # the timed region: the steps alone (no profiling events between launches)
    ms_step, wall = timed(step)
    bu_per_step = len(layouts) * len(ALGOS) * w.b * w.T * w.iters
    value = bu_per_step / (ms_step / 1e3)
    # the same steps with every call on the timing stream, one after another
    ms_serial, _ = timed(step, serial=True)

    # a second pass of the same steps, serial, with HIP events around every
    # launch (library profiling, on the call stream): per-kernel durations
    bi.bi_profile_begin()
    ms_prof, _ = timed(step, serial=True)
    prof = bi.bi_profile_end()
    # a third pass with events around every call: per-call durations, the
    # median over the steps (each step with its own events, one
    # synchronisation at the end, so no call starts on an idle queue)
    step_marks = [{k: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for k in qs}
                  for _ in range(args.steps)]
    torch.cuda.synchronize()
    for marks in step_marks:
        step(marks=marks)
    torch.cuda.synchronize()
    call_ms = {k: statistics.median(m[k][0].elapsed_time(m[k][1]) for m in step_marks) for k in qs}

    # the streaming families ran (soft vectors too: no log-likelihood tensors)
    assert not any(k.startswith("agent") or k == "soft_ll" for k in prof), sorted(prof)
    traffic = {} if args.soft else load_traffic()   # the counters were taken with outcomes
    dense_work = dense_lik_work(w.model, w.obs, soft_np)
    sq_flops, sq_bytes, sq_stored = sparse16_lik_work(w.model, w.obs, soft_np)
    work = {"lik": dense_work, "lik_split": dense_work, "lik_split16": dense_work, "lik_rowcol16": dense_work,
            "lik_sparse": sparse_lik_work(w.model, w.obs, soft_np), "lik_sparse16": (sq_flops, sq_bytes)}
    rooflines = roofline_entries(prof, work, traffic)
    if "lik_sparse16" in rooflines:
        rooflines["lik_sparse16"]["stored_bytes_per_launch"] = sq_stored
    dominant = max(rooflines, key=lambda c: rooflines[c]["total_ms"])
    lik_cls = {"dense": "lik_split" if args.dense_f32 else "lik_rowcol16",
               "sparse": "lik_sparse" if args.sparse_f64 else "lik_sparse16"}
    calls = {}
    for (lay, a), ms in call_ms.items():
        cls = lik_cls[lay]
        nb = work[cls][1] * w.iters
        calls[f"{lay}/{a}"] = {"ms": ms, "algorithmic_bytes": nb, "algorithmic_GBps": nb / (ms / 1e3) / 1e9,
                               "hbm_frac": nb / (ms / 1e3) / 1e9 / PEAK_HBM_GBPS,
                               "belief_updates_per_s": w.b * w.T * w.iters / (ms / 1e3)}
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "belief_updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32+f64" if args.dense_f32 and args.sparse_f64 else "f16x2+f64",
        "data": "synthetic",
        "config": {"workload": "shared model F=4x32 states (U=4), M=4x32 outcomes on all factors, 90% zeros, "
                               "b=64, T=16, 16 iters; step = VMP + MMP on the dense ("
                               + ("fp32 MFMA" if args.dense_f32 else "fp16-pair MFMA") + ") and sparse ("
                               + ("fp64 gathers" if args.sparse_f64 else "fp16-pair MFMA from the nonzeros")
                               + ") A layouts"
                               + ("; soft observation vectors (every outcome weighted, 0.7 on the drawn one)"
                                  if args.soft else ""),
                   "b": w.b, "T": w.T, "iters": w.iters, "algos": list(ALGOS), "layouts": layouts},
        "roofline": rooflines[dominant],
        "roofline_all": rooflines,
        "settle_steps": SETTLE_STEPS,
        "concurrency": "each layout's calls (VMP, then MMP) on a stream of its own, the two layouts' streams "
                       "overlapping inside a step" if len(layouts) > 1 and not args.serial else "one stream",
        "serial": {"ms_per_step": ms_serial, "value": bu_per_step / (ms_serial / 1e3), "unit": "belief_updates/s",
                   "note": "the same step with every call on one stream, one after another"},
        "kernel_timing": "a second pass of the same steps with HIP events around every launch on the call "
                         f"stream ({ms_prof:.3f} ms per step with them); the timed region has none",
        "kernels": {k: {"launches": n, "avg_ms": ms / max(n, 1)} for k, (n, ms) in prof.items()},
        "calls": calls,
        "call_hbm_frac": {k: v["hbm_frac"] for k, v in calls.items()},
        "wall_s_timed": wall,
        "dtype_note": ("dense layout: fp32 matrix-core contractions (v_mfma_f32_16x16x4f32)" if args.dense_f32 else
                       "dense layout: slices as fp16 (high, residual) pairs in 32x32 blocks, 22 significant bits, "
                       "each block read once and contracted towards its rows and its columns with three fp16 "
                       "matrix-core products per fp32 product (v_mfma_f32_16x16x32_f16), fp32 accumulation") + " with fp64 message sums, transitions and softmax; sparse layout: "
                      + ("fp64 throughout" if args.sparse_f64 else
                         "the nonzeros as fp16 pairs, scattered into LDS blocks and contracted with the same "
                         "three-product fp16 matrix-core chains"),
    }
    # the same step captured once in a HIP graph and replayed (the calls only
    # enqueue kernels): launch overhead out of the way; reported beside the
    # eager step above, which stays the headline
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):   # captured on torch's capture stream (st=None: the current one)
        step(None)
    graph.replay()
    torch.cuda.synchronize()
    g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    g0.record(stream)
    for _ in range(args.steps):
        graph.replay()
    g1.record(stream)
    torch.cuda.synchronize()
    g_ms = g0.elapsed_time(g1) / args.steps
    out["graph_replay"] = {"ms_per_step": g_ms, "value": bu_per_step / (g_ms / 1e3), "unit": "belief_updates/s"}
    del graph
    results = {("main", k): v.cpu().numpy() for k, v in qs.items()}

    # what the precision classes buy: the same step with the other class on
    # each layout (fp32 matrix cores on the fp32 copy; fp64 sparse gathers)
    if not args.no_variants and not (args.dense_f32 and args.sparse_f64):
        vp, vq, vw = setup(plain)
        vstep = make_step(vp, vq, vw)
        for _ in range(max(1, args.warmup)):
            vstep()
        v_ms, _ = timed(vstep)
        out["precision_variant"] = {
            "dtype": "f32+f64", "ms_per_step": v_ms, "value": bu_per_step / (v_ms / 1e3), "unit": "belief_updates/s",
            "note": "dense layout on fp32 matrix cores (fp32 slice copy), sparse layout on fp64 gathers"}
        results.update({("variant", k): v.cpu().numpy() for k, v in vq.items()})

    # the oracle timed on the host cores; its outputs on those sampled agents
    # (the same for both layouts) give max |gpu - oracle| of every call
    out["max_abs_err"] = None
    if args.soft:
        # the oracle forms every context's expected log-likelihood again in
        # every iteration (32 slices per entry, 34 G logarithms per agent and
        # call: an estimated 12 minutes on one core), so no bounded sample
        # exists; the soft streaming path's parity is in the GPU tests
        out["cpu_baseline"] = None
        out["cpu_baseline_note"] = ("not timed with soft vectors on this model (an oracle call: an estimated "
                                    "12 minutes per agent)")
    elif not args.no_cpu_baseline:
        base, refs, agents = cpu_baseline(w, list(ALGOS), keep=True)
        out["cpu_baseline"] = base
        out["cpu_baseline_1thread"] = cpu_baseline_1thread(w, "vmp")
        err = {}
        for (kind, (lay, a)), q in results.items():
            if a in refs:
                err[f"{kind}:{lay}/{a}"] = float(np.abs(q[agents] - refs[a]).max())
        main = [v for k, v in err.items() if k.startswith("main:")]
        out["max_abs_err"] = {"value": max(main) if main else None, "per_call": err,
                              "agents": [int(x) for x in agents], "tolerance": 1e-5,
                              "within": bool(main) and max(main) <= 1e-5}
    print(json.dumps(out), flush=True)


def roofline_entries(prof, work, traffic):
    rooflines = {}
    for cls, (kname, src) in LIK.items():
        if cls not in prof:
            continue
        launches, total_ms = prof[cls]
        avg_ms = total_ms / max(launches, 1)
        flops, alg_bytes = work[cls]
        tr = traffic.get(kname)
        hbm = tr["hbm_bytes_per_launch"] if tr and tr.get("kernel_source_sha") == source_sha(src) else None
        if cls in ("lik_split16", "lik_sparse16", "lik_rowcol16"):
            # memory bound: the fp16 products (3 per fp32 product) take a
            # fraction of the time the slice bytes (dense: every entry, 4 B;
            # sparse: the nonzeros, 8 B) do
            bound, peak, unit = "hbm", PEAK_HBM_GBPS, "GB/s"
            achieved = alg_bytes / (avg_ms / 1e3) / 1e9
        else:
            bound, peak = ("mfma", PEAK_FP32_MFMA_TFLOPS) if cls in ("lik", "lik_split") else ("alu", PEAK_FP64_VALU_TFLOPS)
            unit = "TFLOP/s"
            achieved = flops / (avg_ms / 1e3) / 1e12
        rooflines[cls] = {
            "bound": bound, "achieved": achieved, "peak": peak, "unit": unit, "frac": achieved / peak,
            "traffic": hbm, "kernel": kname, "avg_launch_ms": avg_ms, "launches": launches,
            "total_ms": total_ms, "algorithmic_flops_per_launch": flops,
            "algorithmic_bytes_per_launch": alg_bytes,
            "algorithmic_GBps": alg_bytes / (avg_ms / 1e3) / 1e9,
            "measured_hbm_GBps": None if hbm is None else hbm / (avg_ms / 1e3) / 1e9,
            "hbm_frac": None if hbm is None else hbm / (avg_ms / 1e3) / 1e9 / PEAK_HBM_GBPS,
        }
        if cls in ("lik_split16", "lik_sparse16", "lik_rowcol16"):
            f16 = 3 * flops / (avg_ms / 1e3) / 1e12
            rooflines[cls]["fp16_mfma"] = {"achieved_TFLOPs": f16, "peak": PEAK_FP16_MFMA_TFLOPS,
                                           "frac": f16 / PEAK_FP16_MFMA_TFLOPS}
    return rooflines


def cache_probe(torch, dev):
    """Apparent copy bandwidth against working-set size: a device-to-device
    copy of n MiB read plus n MiB written, after three warm-up copies, timed
    with HIP events."""
    res = {}
    for mb in (32, 64, 96, 128, 192, 256, 384, 512, 1024, 2048):
        n = mb * (1 << 20) // 4
        x = torch.ones(n, device=dev)
        y = torch.empty_like(x)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = max(5, 4096 // mb)
        e0.record()
        for _ in range(reps):
            y.copy_(x)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        res[2 * mb] = 2 * mb * (1 << 20) / (ms / 1e3) / 1e9
        del x, y
    print(json.dumps({"copy_working_set_MiB_to_GBps": res}), flush=True)


def bench_sweep(args, bi, synth, torch, dev):
    """The seeded POMDP sweep (770 specs per dimension regime, one model shared
    by 256 agents, T from the spec, 16 iterations): each model packed once with
    every kernel family allowed (BI_SPARSE_A | BI_FAST_F32 | BI_F16_PAIRS),
    FPI, VMP and MMP each timed as the selector routes them (median of
    args.steps calls after args.warmup, HIP events around each call).  value =
    belief updates of all calls / their summed median times.  The oracle
    checks agents 0 and 255 of every call (max-abs error reported)."""
    import numpy as np
    import oracle
    lo, hi = (int(x) for x in args.cases.split(":"))
    regimes = [r for r in args.regimes.split(",") if r]
    flags = bi.BI_SPARSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS
    stream = torch.cuda.current_stream()
    total_bu, total_ms, err, per_algo, fams = 0, 0.0, 0.0, {}, {}
    orc_bu, orc_s = 0, 0.0
    worst = None
    t0 = time.perf_counter()
    n_models = 0
    for regime in regimes:
        for case in range(lo, hi):
            w = synth.sweep_model(case, regime=regime)
            pm = bi.PackedModel(w.model, flags=flags, device=dev)
            obs = torch.from_numpy(w.obs).to(dev)
            act = torch.from_numpy(w.act).to(dev)
            q = torch.empty((w.b, w.T, w.model.n_total), dtype=torch.float32, device=dev)
            for algo in ("fpi", "vmp", "mmp"):
                ws = pm.workspace(w.b, w.T, algo)
                fam = pm.path(w.b, w.T, algo)
                for _ in range(max(1, args.warmup)):
                    pm.infer(algo, obs, act, w.iters, q=q, ws=ws, stream=stream)
                times = []
                for _ in range(args.steps):
                    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    e0.record(stream)
                    pm.infer(algo, obs, act, w.iters, q=q, ws=ws, stream=stream)
                    e1.record(stream)
                    e1.synchronize()
                    times.append(e0.elapsed_time(e1))
                ms = float(np.median(times))
                bu = w.b * w.T * w.iters
                total_bu += bu
                total_ms += ms
                pa = per_algo.setdefault(algo, [0, 0.0])
                pa[0] += bu
                pa[1] += ms
                fams[f"{algo}:{fam}"] = fams.get(f"{algo}:{fam}", 0) + 1
                o0 = time.perf_counter()
                ref = oracle.infer(algo, w.model, w.obs, w.act, w.iters, agents=[0, w.b - 1])
                orc_s += time.perf_counter() - o0
                orc_bu += 2 * w.T * w.iters
                e = float(np.abs(q.cpu().numpy()[[0, w.b - 1]] - ref).max())
                if e > err:
                    err, worst = e, f"{regime} {case} {algo} ({fam})"
            pm.close()
            n_models += 1
            if n_models % 50 == 0:
                print(f"[sweep] {n_models} models, {time.perf_counter() - t0:.0f} s", file=sys.stderr, flush=True)
    out = {
        "metric": METRIC, "value": total_bu / (total_ms / 1e3), "unit": "belief_updates/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": total_ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "per family (f64 agent, f16x2/f32+f64 streaming)",
        "data": "synthetic",
        "config": {"workload": f"seeded POMDP sweep, regimes {regimes}, specs {lo}:{hi} each, b=256, T per spec, "
                               "16 iters, FPI + VMP + MMP as the selector routes them",
                   "models": n_models, "b": 256, "iters": 16},
        "per_algo": {a: {"belief_updates": v[0], "ms": v[1], "value": v[0] / (v[1] / 1e3)} for a, v in per_algo.items()},
        "families": fams,
        "max_abs_err": {"value": err, "worst": worst, "agents": [0, 255], "tolerance": 1e-5, "within": err <= 1e-5},
        "wall_s": time.perf_counter() - t0,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = {"value": orc_bu / max(orc_s, 1e-9), "unit": "belief_updates/s", "cores": 2,
                               "kind": "oracle",
                               "sample": f"agents 0 and 255 of every call ({orc_bu} belief updates, one thread per "
                                         f"agent), {orc_s:.1f} s"}
    print(json.dumps(out), flush=True)


def bench_agent(args, bi, synth, torch, dev):
    """One step = one call of the workload's algorithm over its whole batch
    (online workloads: T one-step calls and T - 1 predictive priors)."""
    import numpy as np
    cfg, algo, opts = AGENT_WORKLOADS[args.workload]
    w = getattr(synth, cfg)(bdeps=synth.THREE_FACTOR_BDEPS) if opts.get("bdeps") else getattr(synth, cfg)()
    rolling = bool(opts.get("rolling"))
    if rolling and args.soft:
        print("bench.py: --soft is not combined with the online workload", file=sys.stderr)
        sys.exit(2)
    pm = bi.PackedModel(w.model, flags=bi.BI_DENSE_A, device=dev)
    obs = torch.from_numpy(w.obs).to(dev)
    act = torch.from_numpy(w.act).to(dev)
    q = torch.empty((w.b, w.T, w.model.n_total), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    assert pm.workspace(w.b, w.T, algo) is None, "per-agent workloads run on the agent-resident kernels"
    soft_np = None
    if args.soft:
        import numpy as np
        soft_np = synth.soft_obs(np.random.Generator(np.random.PCG64(17855)), w.obs, w.model.K, confidence=0.7)
        soft_dev = torch.from_numpy(soft_np).to(dev)
        ws = pm.workspace_soft(w.b, w.T, algo)

    if rolling:
        # per step t: its observations, its own output, the prior of step t + 1
        obs_t = [obs[:, t:t + 1].contiguous() for t in range(w.T)]
        act_t = [act[:, t].contiguous() for t in range(w.T - 1)]
        q_t = [torch.empty((w.b, 1, w.model.n_total), dtype=torch.float32, device=dev) for _ in range(w.T)]
        priors = [torch.empty((w.b, w.model.n_total), dtype=torch.float32, device=dev) for _ in range(2)]

    def step():
        if rolling:
            prior = None   # step 0: D of the packed model
            for t in range(w.T):
                pm.infer(algo, obs_t[t], None, w.iters, q=q_t[t], stream=stream, prior=prior)
                if t + 1 < w.T:
                    prior = pm.predict(q_t[t][:, 0], act_t[t], out=priors[t % 2], stream=stream)
        elif soft_np is not None:
            pm.infer_soft(algo, soft_dev, act, w.iters, q=q, ws=ws, stream=stream)
        else:
            pm.infer(algo, obs, act, w.iters, q=q, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    def timed():
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ev0.record(stream)
        for _ in range(args.steps):
            step()
        ev1.record(stream)
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) / args.steps, time.perf_counter() - t0

    ms_step, wall = timed()          # the timed region: the steps alone
    bi.bi_profile_begin()            # a second pass with HIP events around every launch
    timed()
    prof = bi.bi_profile_end()
    bu = w.b * w.T * w.iters
    cls = next(k for k in ("agent_filter_tile", "agent_filter", "agent_window_tile", "agent_window") if k in prof)
    launches, total_ms = prof[cls]
    avg_ms = total_ms / max(launches, 1)
    fl, nb = agent_work(w.model, w.T, algo)
    t_launch = 1 if rolling else w.T   # steps per launch
    flops = fl * w.b * t_launch * w.iters
    achieved = flops / (avg_ms / 1e3) / 1e12
    out = {
        "metric": METRIC, "value": bu / (ms_step / 1e3), "unit": "belief_updates/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"{w.name}: per-agent models, {algo.upper()} x{w.iters}"
                               + (", soft observations" if soft_np is not None else "")
                               + (", online (one step per call, predictive prior carried)" if rolling else "")
                               + (f", B-dependency lists {w.model.bdeps}" if w.model.bdeps else ""),
                   "b": w.b, "T": w.T, "iters": w.iters, "algos": [algo], "soft": soft_np is not None,
                   "rolling": rolling},
        "roofline": None,
        "kernels": {k: {"launches": n, "avg_ms": ms / max(n, 1)} for k, (n, ms) in prof.items()},
        "wall_s_timed": wall,
    }
    # Both rooflines of the agent kernel: the fp64 arithmetic, and the bytes
    # of one read of the observed fp64 slices per belief update (its counted
    # traffic from profiles/traffic_agent.json while the kernel source is
    # unchanged).  The counters show the kernel waiting on memory, not on
    # arithmetic; the headline roofline is the one it is closer to.
    alg_bytes = nb * w.b * t_launch * w.iters
    tr = load_agent_traffic().get(args.workload)
    hbm = tr["hbm_bytes_per_launch"] if tr and tr.get("kernel_source_sha") == source_sha("agent.hip") else None
    gbps = alg_bytes / (avg_ms / 1e3) / 1e9
    out["roofline_all"] = {
        "hbm": {"bound": "hbm", "achieved": gbps, "peak": PEAK_HBM_GBPS, "unit": "GB/s", "frac": gbps / PEAK_HBM_GBPS,
                "traffic": hbm, "kernel": cls + "_kernel", "avg_launch_ms": avg_ms, "launches": launches,
                "algorithmic_bytes_per_launch": alg_bytes,
                "measured_hbm_GBps": None if hbm is None else hbm / (avg_ms / 1e3) / 1e9},
        "alu": {"bound": "alu", "achieved": achieved, "peak": PEAK_FP64_VALU_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / PEAK_FP64_VALU_TFLOPS, "traffic": hbm, "kernel": cls + "_kernel",
                "avg_launch_ms": avg_ms, "launches": launches, "algorithmic_flops_per_launch": flops}}
    out["roofline"] = max(out["roofline_all"].values(), key=lambda r: r["frac"])
    if soft_np is not None:
        sl, sms = prof["soft_ll"]
        s_avg = sms / max(sl, 1)
        s_bytes = soft_ll_bytes(w.model, w.b, w.T)
        s_ach = s_bytes / (s_avg / 1e3) / 1e9
        out["roofline_all"].update({
            "soft_ll": {"bound": "hbm", "achieved": s_ach, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                        "frac": s_ach / PEAK_HBM_GBPS, "traffic": None, "kernel": "soft_ll_kernel",
                        "avg_launch_ms": s_avg, "launches": sl, "algorithmic_bytes_per_launch": s_bytes}})
        if s_avg > avg_ms:
            out["roofline"] = out["roofline_all"]["soft_ll"]
    out["max_abs_err"] = None
    if not args.no_cpu_baseline:
        base, refs, agents = cpu_baseline(w, [algo], soft=soft_np, keep=True)
        out["cpu_baseline"] = base
        out["cpu_baseline_1thread"] = cpu_baseline_1thread(w, algo)
        if not rolling:
            e = float(np.abs(q.cpu().numpy()[agents] - refs[algo]).max())
            out["max_abs_err"] = {"value": e, "agents": [int(x) for x in agents], "tolerance": 1e-5,
                                  "within": e <= 1e-5}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
