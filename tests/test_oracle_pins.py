"""The oracle against results the paper and mathematics fix (CPU only)."""
import pytest

import oracle
from oracle_pins import ALL_PINS


@pytest.mark.parametrize("name", sorted(ALL_PINS))
def test_pin(name):
    fn, tol = ALL_PINS[name]
    err = fn(oracle.infer)
    assert err <= tol, f"{name}: max deviation {err:.3e} > {tol:.1e}"


def test_rejects_bad_arguments():
    import numpy as np
    from paper_2607_17855_amd import synth
    w = synth.random_small(1, b=2)
    with pytest.raises(ValueError):
        oracle.infer("vmp", w.model, w.obs, w.act, 0)
    bad = synth.Model(w.model.n, w.model.U, w.model.K, [[len(w.model.n)]] + w.model.deps[1:], w.model.mb,
                      w.model.A, w.model.B, w.model.D)
    with pytest.raises(ValueError):
        oracle.infer("vmp", bad, w.obs, w.act, 2)
    assert np.all(np.isfinite(oracle.infer("mmp", w.model, w.obs, w.act, 2)))
    for tau in (0.0, -0.5, 1.5):
        with pytest.raises(ValueError):
            oracle.infer("vmp", w.model, w.obs, w.act, 2, damping=tau)
