"""The test-side statement of the paged-cache layout (tests/cache_layout.py)
against the byte formula of the header, element by element (no GPU)."""
import numpy as np
import pytest

from cache_layout import from_cache, piece_bytes, to_cache


@pytest.mark.parametrize("R", [48, 36, 72, 30, 24, 16, 13, 1])
def test_cache_layout_formula(R):
    rng = np.random.default_rng(R)
    nb, H, bs = 3, 2, 7
    rec = rng.integers(0, 256, (nb, H, bs, R), dtype=np.uint8)
    cache = to_cache(rec)
    P = piece_bytes(R)
    assert R % P == 0 and (P == 16 or R % (2 * P) != 0) and (P in (8, 16) or P == R)
    flat = cache.reshape(nb, H, bs * R)
    for b in range(nb):
        for h in range(H):
            for s in range(bs):
                for k in range(R):
                    j, o = divmod(k, P)
                    assert flat[b, h, (j * bs + s) * P + o] == rec[b, h, s, k]
    np.testing.assert_array_equal(from_cache(cache), rec)
