"""Calls on two streams at once (the throughput step runs the dense and the
sparse layouts' calls this way): every call's output equals, bit for bit,
the same call run alone.  The calls share no workspace; each stream runs
its calls in order."""
import os

import numpy as np
import pytest

from paper_2607_17855_amd import bi, synth

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    return torch


def _shared(seed, n, K, b, T, sparsity):
    rng = np.random.Generator(np.random.PCG64(seed))
    model = synth.make_model(rng, n, [2, 1, 2, 1], K, [[0, 1, 2, 3]] * len(K), 1, 1.0, 1.0, sparsity=sparsity,
                             uniform_D=False)
    obs, act = synth.sample_sequences(rng, model, b, T)
    return synth.Workload(f"conc{seed}", ["vmp", "mmp"], model, obs, act, 4)


def test_layouts_on_two_streams_match_serial():
    torch = _torch()
    old = os.environ.pop("BI_FORCE_PATH", None)
    cases = {
        "dense": (_shared(3100, [12, 32, 2, 32], [4, 2], 40, 4, 0.0), bi.BI_DENSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS),
        "sparse": (_shared(3101, [6, 16, 4, 32], [3, 2], 24, 5, 0.8),
                   bi.BI_SPARSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS),
    }
    pms = {k: bi.PackedModel(w.model, fl) for k, (w, fl) in cases.items()}
    try:
        dev = {k: tuple(torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in (w.obs, w.act))
               for k, (w, _) in cases.items()}
        keys = [(k, a) for k in cases for a in ("vmp", "mmp")]
        fam = {"dense": "stream", "sparse": "sparse"}   # the families the throughput step runs
        ws = {}
        for k, a in keys:
            w = cases[k][0]
            os.environ["BI_FORCE_PATH"] = fam[k]
            assert pms[k].path(w.b, w.T, a) == fam[k]
            ws[(k, a)] = pms[k].workspace(w.b, w.T, a)
        q = {key: torch.empty((cases[key[0]][0].b, cases[key[0]][0].T, cases[key[0]][0].model.n_total),
                              dtype=torch.float32, device="cuda") for key in keys}

        def call(k, a, st):
            w = cases[k][0]
            os.environ["BI_FORCE_PATH"] = fam[k]   # read by the host when the call is issued
            pms[k].infer(a, dev[k][0], dev[k][1], w.iters, q=q[(k, a)], ws=ws[(k, a)], stream=st)

        for k, a in keys:
            call(k, a, torch.cuda.current_stream())
        torch.cuda.synchronize()
        ref = {key: v.cpu().numpy() for key, v in q.items()}
        side = {k: torch.cuda.Stream() for k in cases}
        main = torch.cuda.current_stream()
        for rep in range(3):
            print(f"[gpu] two streams, pass {rep}", flush=True)
            for v in q.values():
                v.fill_(-1.0)
            fork = torch.cuda.Event()
            fork.record(main)
            for k in cases:
                side[k].wait_event(fork)
                for a in ("vmp", "mmp"):
                    call(k, a, side[k])
            for k in cases:
                join = torch.cuda.Event()
                join.record(side[k])
                main.wait_event(join)
            torch.cuda.synchronize()
            for key in keys:
                assert np.array_equal(q[key].cpu().numpy(), ref[key]), key
    finally:
        for pm in pms.values():
            pm.close()
        os.environ.pop("BI_FORCE_PATH", None)
        if old is not None:
            os.environ["BI_FORCE_PATH"] = old
