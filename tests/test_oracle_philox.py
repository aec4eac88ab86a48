"""Pins for the oracle's counter-based generator and its dropout masks.

Philox4x32-10 against the known-answer vectors published with the
generator's reference implementation (Salmon et al., SC'11, Random123), the
mask's element/counter/word mapping against a scalar recomputation, and the
keep rate, step and seed dependence against what a uniform 24-bit draw
implies."""
import numpy as np
import pytest

from oracle import philox


@pytest.mark.parametrize("ctr,key,out", [
    ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF,) * 4, (0xFFFFFFFF, 0xFFFFFFFF), (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
])
def test_philox4x32_10_known_answers(ctr, key, out):
    got = philox.philox4x32(*[np.array([c]) for c in ctr], *key)
    assert tuple(int(w[0]) for w in got) == out


def _scalar_philox(c, k):
    """Plain-integer Philox4x32-10, one counter (a second transcription of the
    round, with Python integers instead of uint64 arrays)."""
    c, k = list(c), list(k)
    for r in range(10):
        if r:
            k = [(k[0] + 0x9E3779B9) % 2 ** 32, (k[1] + 0xBB67AE85) % 2 ** 32]
        p0, p1 = 0xD2511F53 * c[0], 0xCD9E8D57 * c[2]
        c = [(p1 >> 32) ^ c[1] ^ k[0], p1 % 2 ** 32, (p0 >> 32) ^ c[3] ^ k[1], p0 % 2 ** 32]
    return c


def test_mask_indexing_matches_scalar_recomputation():
    n, f, p, seed, step = 3, 20, 0.3, 0x123456789ABCDEF0, 2 ** 32 + 5
    keep = philox.dropout_keep(seed, step, n, f, p)
    thresh, _ = philox.dropout_params(p)
    for i in range(n * f):
        q = i // 4
        x = _scalar_philox((q % 2 ** 32, q >> 32, step % 2 ** 32, step >> 32), (seed % 2 ** 32, seed >> 32))[i % 4]
        assert keep[i // f, i % f] == ((x >> 8) >= thresh), i


@pytest.mark.parametrize("p", [0.1, 0.2, 0.3])
def test_keep_rate(p):
    n, f = 2048, 512
    keep = philox.dropout_keep(7, 11, n, f, p)
    thresh, scale = philox.dropout_params(p)
    q = 1.0 - thresh / 2.0 ** 24
    sigma = np.sqrt(q * (1 - q) / keep.size)
    assert abs(keep.mean() - q) < 5 * sigma
    assert abs(q - (1 - p)) < 2.0 ** -23
    assert scale == np.float32(1.0 / (1.0 - np.float64(np.float32(p))))


def test_masks_differ_by_step_and_seed_and_are_uncorrelated():
    n, f, p = 512, 512, 0.5
    a = philox.dropout_keep(1, 0, n, f, p).astype(np.float64).ravel()
    b = philox.dropout_keep(1, 1, n, f, p).astype(np.float64).ravel()
    c = philox.dropout_keep(2, 0, n, f, p).astype(np.float64).ravel()
    for u, v in ((a, b), (a, c), (b, c)):
        r = np.corrcoef(u, v)[0, 1]
        assert abs(r) < 5 / np.sqrt(u.size)
    # neighbouring features (same counter, different output words) too
    m = philox.dropout_keep(3, 4, n, f, p).astype(np.float64)
    r = np.corrcoef(m[:, 0::2].ravel(), m[:, 1::2].ravel())[0, 1]
    assert abs(r) < 5 / np.sqrt(m.size / 2)


def test_rate_zero_keeps_everything_and_bad_rates_raise():
    assert philox.dropout_keep(5, 5, 4, 8, 0.0).all()
    assert philox.dropout_params(0.0) == (0, 1.0)
    for bad in (-0.1, 1.0, 1.5):
        with pytest.raises(ValueError):
            philox.dropout_params(bad)
