"""The parity tests' own error measures, checked on the CPU against planted mistakes (the mistakes
are planted in an oracle result, never in the HIP path)."""
import numpy as np

import oracle
import synth
from tests.helpers import rel_fro, tile_rel_errors


def _ns(m, n, seed):
    rng = np.random.default_rng(seed)
    x = synth.f32_to_bf16_bits(rng.standard_normal((m, n), dtype=np.float32))
    return oracle.newton_schulz(x, *synth.NS_COEFFS, 5)


def test_block_errors_flag_one_misplaced_block_that_the_global_error_misses():
    O = _ns(1024, 4096, 3)       # 4 x 16 blocks of 256 x 256
    bad = O.copy()
    bad[256:512, 768:1024] = O[256:512, 768:1024].T  # one block stored transposed
    assert rel_fro(bad, O) < 2e-1                      # diluted over 64 blocks ...
    t = tile_rel_errors(bad, O)
    assert t.shape == (4, 16)
    assert t[1, 3] > 1.0 and np.all(np.delete(t.ravel(), 1 * 16 + 3) == 0.0)  # ... but not per block


def test_block_errors_of_a_uniform_perturbation_equal_the_global_error():
    O = _ns(512, 768, 4)
    bad = O * (1 + 1e-2)
    t = tile_rel_errors(bad, O)
    assert np.allclose(t, 1e-2, rtol=1e-9) and abs(rel_fro(bad, O) - 1e-2) < 1e-12


def test_block_errors_on_ragged_edges():
    O = _ns(300, 129, 5)           # edge blocks partial in both directions
    bad = O.copy()
    bad[-1, -1] += 1.0
    t = tile_rel_errors(bad, O)
    assert t.shape == (2, 1) and t[1, 0] > 0 and t[0, 0] == 0
