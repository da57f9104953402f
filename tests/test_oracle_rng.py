"""The oracle's counter-based generator (Philox4x32-10) and its 16-bit draws.

No known-answer vectors for Philox4x32-10 are available offline, so the raw
bit stream is "parity unpinned" against external data. What is pinned here:
  * invertibility: running the published round structure backwards (the
    inverse of multiplication by an odd constant mod 2^32, computed by Newton
    iteration) recovers the counter from the oracle's output, for random
    keys and counters; a wrong multiplier, key constant or word order in the
    oracle breaks this;
  * the draw layout (counter = (i/8, t, k, 0), 16-bit halves in order);
  * statistics: uniform 16-bit draws, balanced bits, no correlation between
    neighbouring counters.
"""
import numpy as np
import pytest

from oracle import ref

MASK = 0xFFFFFFFF
M0, M1 = 0xD2511F53, 0xCD9E8D57
W0, W1 = 0x9E3779B9, 0xBB67AE85


def inv_odd(a):
    """Inverse of odd a modulo 2^32 by Newton iteration x <- x (2 - a x)."""
    x = a  # correct to 3 bits for odd a
    for _ in range(5):
        x = (x * (2 - a * x)) & MASK
    assert (a * x) & MASK == 1
    return x


def philox_inverse(key, out, rounds=10):
    k0s, k1s = [key[0] & MASK], [key[1] & MASK]
    for _ in range(rounds - 1):
        k0s.append((k0s[-1] + W0) & MASK)
        k1s.append((k1s[-1] + W1) & MASK)
    iM0, iM1 = inv_odd(M0), inv_odd(M1)
    y = [int(v) for v in out]
    for r in reversed(range(rounds)):
        x2 = (y[1] * iM1) & MASK          # lo1 = M1 * x2
        x0 = (y[3] * iM0) & MASK          # lo0 = M0 * x0
        hi1 = (M1 * x2) >> 32
        hi0 = (M0 * x0) >> 32
        x1 = y[0] ^ hi1 ^ k0s[r]
        x3 = y[2] ^ hi0 ^ k1s[r]
        y = [x0, x1, x2, x3]
    return y


def test_philox_output_inverts_to_counter():
    rng = np.random.default_rng(0)
    for _ in range(200):
        key = [int(v) for v in rng.integers(0, 2 ** 32, 2)]
        ctr = [int(v) for v in rng.integers(0, 2 ** 32, 4)]
        out = ref.philox4x32_10(key, ctr)
        assert philox_inverse(key, out) == ctr
    # distinct counters -> distinct outputs (a bijection), and every key matters
    a = ref.philox4x32_10([1, 2], [0, 0, 0, 0])
    assert not np.array_equal(a, ref.philox4x32_10([1, 2], [1, 0, 0, 0]))
    assert not np.array_equal(a, ref.philox4x32_10([1, 3], [0, 0, 0, 0]))
    assert not np.array_equal(a, ref.philox4x32_10([2, 2], [0, 0, 0, 0]))


def test_draw_layout():
    seed = (0xABCDEF01 << 32) | 0x12345678
    for (k, t, i) in [(0, 1, 0), (3, 17, 5), (1023, 1008, 1007), (7, 4000, 3999)]:
        x = ref.philox4x32_10([seed & MASK, seed >> 32], [i // 8, t, k, 0])
        j = i % 8
        want = (int(x[j // 2]) >> (16 * (j % 2))) & 0xFFFF
        assert ref.draw(seed, k, t, i) == want
    # the 8 draws of one counter are the 8 halves of its output
    x = ref.philox4x32_10([5, 0], [2, 9, 4, 0])
    halves = [(int(x[j // 2]) >> (16 * (j % 2))) & 0xFFFF for j in range(8)]
    assert [ref.draw(5, 4, 9, 16 + j) for j in range(8)] == halves


def test_draws_uniform_and_balanced():
    vals = np.array([ref.draw(99, k, t, i) for k in range(4) for t in range(1, 60) for i in range(t)],
                    dtype=np.int64)
    m = vals.size
    # chi-square on the top 6 bits (64 bins): mean 63, sd ~11.2
    counts = np.bincount(vals >> 10, minlength=64)
    exp = m / 64
    chi2 = float(((counts - exp) ** 2 / exp).sum())
    assert chi2 < 63 + 6 * np.sqrt(2 * 63)
    for b in range(16):
        ones = int(((vals >> b) & 1).sum())
        assert abs(ones - m / 2) < 5 * np.sqrt(m / 4)
    # neighbouring draws are uncorrelated
    a = vals[:-1].astype(np.float64) - 32767.5
    c = vals[1:].astype(np.float64) - 32767.5
    corr = float((a * c).mean() / np.sqrt((a * a).mean() * (c * c).mean()))
    assert abs(corr) < 5 / np.sqrt(m)
