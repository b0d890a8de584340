"""Host-side paging of the KV caches used by the paged-cache GPU tests and bench."""
import numpy as np

from paper_2605_31457_amd import step as S


def test_paged_cache_layout_round_trip():
    """The host-side paging helper places row s of sequence b in block table[b, s // P]."""
    rng = np.random.default_rng(0)
    K = rng.standard_normal((3, 2, 70, 8)).astype(np.float32)
    V = rng.standard_normal((3, 2, 70, 8)).astype(np.float32)
    Kp, Vp, table = S.paged_cache(K, V, 16, seed=5)
    assert table.shape == (3, 5) and len(set(table.ravel())) == 15
    for b in range(3):
        for s in range(70):
            np.testing.assert_array_equal(Kp[table[b, s // 16], :, s % 16], K[b, :, s])
            np.testing.assert_array_equal(Vp[table[b, s // 16], :, s % 16], V[b, :, s])
