"""The seeded input generators (no inference arithmetic): shapes and the
distribution properties the tests rely on."""
import numpy as np

from paper_2607_17855_amd import synth


def test_random_prior_blocks_are_distributions_with_zeros():
    rng = np.random.Generator(np.random.PCG64(5))
    n = [3, 1, 7, 40]
    p = synth.random_prior(rng, n, 50, alpha=0.7, p_zero=0.4)
    assert p.shape == (50, sum(n)) and p.dtype == np.float32
    offs = np.cumsum([0] + n)
    for f in range(len(n)):
        blk = p[:, offs[f]:offs[f + 1]].astype(np.float64)
        assert blk.min() >= 0.0
        assert np.abs(blk.sum(1) - 1.0).max() < 1e-6
        assert (blk > 0).any(axis=1).all()           # one state of every block kept
    assert (p[:, offs[3]:] == 0).any()               # zeros do occur
    q = synth.random_prior(np.random.Generator(np.random.PCG64(5)), n, 50, alpha=0.7, p_zero=0.4)
    assert np.array_equal(p, q)                      # reproducible from the seed
