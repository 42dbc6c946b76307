"""Host-side checks of arithmetic identities the kernels rely on (no GPU).

The rANS chunk coder divides its 32-bit state by a symbol frequency f in
[1, 4096] with a per-symbol reciprocal instead of a divide (Granlund and
Montgomery, division by invariant integers): l = ceil(log2 f),
m = floor(2^32 (2^l - f) / f) + 1, t = mulhi(x, m),
x / f = (t + ((x - t) >> min(l, 1))) >> max(l - 1, 0).
Here the identity is checked for every f on the states the coder meets and
at the edges of the 32-bit range."""
import numpy as np


def _recip(f):
    l = (f - 1).bit_length() if f > 1 else 0
    m = ((((1 << l) - f) << 32) // f) + 1
    return m, min(l, 1), max(l - 1, 0)


def test_reciprocal_division_every_frequency():
    rng = np.random.default_rng(12)
    for f in range(1, 4097):
        m, sh1, sh2 = _recip(f)
        assert 0 < m < (1 << 32)
        hi = min(f << 20, 1 << 32)  # states before coding lie in [2^16, f 2^20)
        x = np.concatenate([
            rng.integers(1 << 16, hi, 2000, dtype=np.uint64),
            np.array([0, 1, f - 1, f, f + 1, (1 << 16), hi - 1,
                      (1 << 32) - 1, (1 << 32) - f], dtype=np.uint64),
            np.arange(1, 64, dtype=np.uint64) * np.uint64(f) - np.uint64(1),
        ]) & np.uint64(0xFFFFFFFF)
        t = (x * np.uint64(m)) >> np.uint64(32)
        q = (t + ((x - t) >> np.uint64(sh1))) >> np.uint64(sh2)
        np.testing.assert_array_equal(q, x // np.uint64(f), err_msg=f"f={f}")
