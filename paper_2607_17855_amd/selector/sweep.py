"""Time every eligible kernel family on the sweep models (one GPU).

For each seeded sweep POMDP (uniform and skewed dimension regimes, one model
shared by b agents) and each of VMP / MMP, the model is packed five ways
(dense fp64 planes; plus the fp32 copy for the dense streaming kernels; plus
the sparse planes; the fp16-pair copy (BI_F16_PAIRS) for the dense streaming
kernels, "stream16"; the sparse fp16-pair layout, "sparse16") and the family
each packing is for is timed with BI_FORCE_PATH: median of `--reps` calls after one warm-up, HIP events on
the call stream.  Each family's output is also compared with the
agent-resident fp64 result (max abs difference, recorded).  One JSON line
per (regime, case, algo) goes to --out; progress goes to stdout.

  python -m paper_2607_17855_amd.selector.sweep --regime uniform --cases 0:770 --out sweep.jsonl
"""
import argparse
import json
import os
import statistics
import sys
import time


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--regime", choices=["uniform", "skewed"], default="uniform")
    ap.add_argument("--cases", default="0:770", help="start:stop")
    ap.add_argument("--b", type=int, default=256)
    ap.add_argument("--iters", type=int, default=16)
    ap.add_argument("--reps", type=int, default=3)
    ap.add_argument("--out", required=True)
    args = ap.parse_args()
    import numpy as np
    import torch
    from paper_2607_17855_amd import bi, synth

    lo, hi = (int(x) for x in args.cases.split(":"))
    flags = {"agent": bi.BI_DENSE_A, "stream": bi.BI_DENSE_A | bi.BI_FAST_F32, "sparse": bi.BI_SPARSE_A,
             "stream16": bi.BI_DENSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS,
             "sparse16": bi.BI_SPARSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS}
    force = {"agent": "agent", "stream": "stream", "sparse": "sparse", "stream16": "stream", "sparse16": "sparse"}
    stream = torch.cuda.current_stream()
    t_start = time.time()
    with open(args.out, "a") as out:
        for case in range(lo, hi):
            w = synth.sweep_model(case, b=args.b, regime=args.regime)
            w = synth.Workload(w.name, w.algos, w.model, w.obs, w.act, args.iters)
            obs = torch.from_numpy(w.obs).cuda()
            act = torch.from_numpy(w.act).cuda()
            pms = {k: bi.PackedModel(w.model, fl) for k, fl in flags.items()}
            for algo in ("vmp", "mmp"):
                rec = {"regime": args.regime, "case": case, "algo": algo, "b": w.b, "T": w.T}
                ref = None
                for fam, pm in pms.items():
                    os.environ["BI_FORCE_PATH"] = force[fam]
                    try:
                        if pm.path(w.b, w.T, algo) != force[fam]:
                            continue          # not eligible with this packing
                        q = torch.empty((w.b, w.T, w.model.n_total), dtype=torch.float32, device="cuda")
                        ws = pm.workspace(w.b, w.T, algo)
                        pm.infer(algo, obs, act, w.iters, q=q, ws=ws, stream=stream)
                        times = []
                        for _ in range(args.reps):
                            e0 = torch.cuda.Event(enable_timing=True)
                            e1 = torch.cuda.Event(enable_timing=True)
                            e0.record(stream)
                            pm.infer(algo, obs, act, w.iters, q=q, ws=ws, stream=stream)
                            e1.record(stream)
                            e1.synchronize()
                            times.append(e0.elapsed_time(e1))
                        rec["t_" + fam] = statistics.median(times)
                        qn = q.cpu().numpy()
                        if fam == "agent":
                            ref = qn
                        elif ref is not None:
                            rec["diff_" + fam] = float(np.abs(qn - ref).max())
                    finally:
                        os.environ.pop("BI_FORCE_PATH", None)
                out.write(json.dumps(rec) + "\n")
                out.flush()
            for pm in pms.values():
                pm.close()
            if (case - lo) % 10 == 0 or case == hi - 1:
                print(f"[sweep] {args.regime} case {case} ({time.time() - t_start:.0f} s)", flush=True)


if __name__ == "__main__":
    sys.exit(main())
