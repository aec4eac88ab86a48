"""Counter-based random numbers for dropout masks: Philox4x32-10.

Test infrastructure only (see the package docstring).

Philox4x32 is the counter-based generator of Salmon, Moraes, Dror and Shaw,
"Parallel random numbers: as easy as 1, 2, 3" (SC'11). A 128-bit counter
(four 32-bit words c0..c3) and a 64-bit key (k0, k1) go through R rounds;
each round multiplies c0 and c2 by fixed 32-bit constants, keeps both halves
of the 64-bit products, and mixes them with c1, c3 and the key:

    (hi0, lo0) = M0 * c0,   (hi1, lo1) = M1 * c2
    c <- (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0)

with M0 = 0xD2511F53, M1 = 0xCD9E8D57; between rounds the key is bumped by
the Weyl constants (0x9E3779B9, 0xBB67AE85) modulo 2^32. R = 10 is the
published default. The four words after the last round are the output.

The paper's adaptive regularisation raises the dropout rate with the image
resolution (Sec. 4.1; rates 0.1-0.3 in the schedules of Tables 7 and 9) but
fixes neither the generator nor the placement; here the mask drops features
before the classifier, and keep(n, j) of training step t is defined from this
generator (the same definition the library documents for rn18_set_dropout):

    i = n F + j,  q = i div 4,  counter = (q mod 2^32, q div 2^32,
    t mod 2^32, t div 2^32),  key = (seed mod 2^32, seed div 2^32),
    x = output word i mod 4,  keep iff (x >> 8) >= floor(p 2^24),

and kept features are multiplied by 1 / (1 - p) rounded to float32.
"""
import numpy as np

M0, M1 = 0xD2511F53, 0xCD9E8D57
W0, W1 = 0x9E3779B9, 0xBB67AE85
MASK32 = 0xFFFFFFFF


def philox4x32(c0, c1, c2, c3, k0, k1, rounds=10):
    """Philox4x32-R on arrays of counters (values < 2^32, any integer dtype)
    with a scalar key; returns the four output words as uint64 arrays."""
    c0, c1, c2, c3 = (np.asarray(c, dtype=np.uint64) & np.uint64(MASK32) for c in (c0, c1, c2, c3))
    k0, k1 = int(k0) & MASK32, int(k1) & MASK32
    m0, m1, mask = np.uint64(M0), np.uint64(M1), np.uint64(MASK32)
    for r in range(rounds):
        if r > 0:
            k0 = (k0 + W0) & MASK32
            k1 = (k1 + W1) & MASK32
        p0 = m0 * c0                      # < 2^64: exact in uint64
        p1 = m1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & mask
        hi1, lo1 = p1 >> np.uint64(32), p1 & mask
        c0, c1, c2, c3 = hi1 ^ c1 ^ np.uint64(k0), lo1, hi0 ^ c3 ^ np.uint64(k1), lo0
    return c0, c1, c2, c3


def dropout_params(p):
    """(threshold, scale) of a dropout rate p in [0, 1): the rate is taken as
    the float32 the library receives; threshold = floor(p 2^24) compares with
    the top 24 bits of an output word, scale = float32(1 / (1 - p))."""
    p = float(np.float32(p))
    if not 0.0 <= p < 1.0:
        raise ValueError("dropout rate must be in [0, 1)")
    return int(np.floor(p * 16777216.0)), float(np.float32(1.0 / (1.0 - p)))


def dropout_keep(seed, step, n, f, p):
    """Boolean keep mask [n, f] of training step `step` (definition above)."""
    thresh, _ = dropout_params(p)
    i = np.arange(n * f, dtype=np.uint64)
    q = i >> np.uint64(2)
    step, seed = int(step), int(seed)
    words = philox4x32(q & np.uint64(MASK32), q >> np.uint64(32), np.full_like(q, step & MASK32),
                       np.full_like(q, (step >> 32) & MASK32), seed & MASK32, (seed >> 32) & MASK32)
    x = np.choose((i & np.uint64(3)).astype(np.int64), words)
    return ((x >> np.uint64(8)) >= np.uint64(thresh)).reshape(n, f)
