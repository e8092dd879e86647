"""RRF-NORMAL-v1: the counter-based Gaussian sketch, oracle side.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

The paper fills each sketch block with standard Gaussian values (Alg. 2,
sketch step; cuRAND in the implementation section).  To let a CPU oracle
reproduce the GPU's sketch bit for bit, the sketch is *defined* here as a pure
function of (seed, global column g, row r):

Bits
    Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
    easy as 1, 2, 3", SC'11) with key (seed, domain) and counter
    (q, g, 0, 0).  Counter block q of column g yields rows 4q .. 4q+3.
    Domain 0 is the sketch.  The oracle takes the words from numpy's Philox
    (an independent library implementation); ``philox4x64_10_py`` is a
    from-the-definition implementation used to pin numpy's counter convention.

Uniforms, from one block (w0, w1, w2, w3)
    u1 = ((w0 >> 11) + 1) * 2^-53  in (0, 1]
    u2 = (w1 >> 11) * 2^-53        in [0, 1)
    and likewise (u1', u2') from (w2, w3).

Box--Muller
    rows 4q, 4q+1   = r cos(theta), r sin(theta)  with r = sqrt(-2 ln u1),
                                                   theta = 2 pi u2
    rows 4q+2, 4q+3 = the same from (u1', u2').
    Rows >= n are dropped, so column g does not depend on n beyond its length,
    and the sketch block i is just columns [i b, i b + b_i) of one global
    matrix, so it does not depend on b either.

Transcendental-free ln, sin, cos (binary64 +, -, *, /, sqrt only, each
correctly rounded, no fused multiply-add, in exactly this order)
    ln u:   u = f 2^e with f in [SQRT_HALF, 2 SQRT_HALF) by frexp plus one
            doubling when f < SQRT_HALF; s = (f - 1) / (f + 1); z = s s;
            p = 1/21, then p = p z + 1/(2j+1) for j = 9 .. 0;
            ln u = e LN2 + (s + s) p.
    theta:  t = 4 u2; q = floor(t); phi = (t - q) PIO2; x = phi phi;
            ps = pc = 1, then for k = 11 .. 1:
              ps = 1 - (x ps) S_k     with S_k = 1/((2k)(2k+1))
              pc = 1 - (x pc) C_k     with C_k = 1/((2k-1)(2k))
            sin phi = phi ps, cos phi = pc; rotate by the quadrant q.
    Every coefficient 1/(integer) (1/(2j+1), S_k, C_k) is the correctly
    rounded binary64 quotient, computed once and then multiplied.
    Constants: SQRT_HALF = 0x1.6a09e667f3bcdp-1, LN2 = 0x1.62e42fefa39efp-1,
    PIO2 = 0x1.921fb54442d18p+0 (the binary64 values nearest sqrt(1/2),
    ln 2 and pi/2).

Precision
    The float32 sketch is the float64 value rounded to nearest-even.
"""

import numpy as np

SQRT_HALF = float.fromhex("0x1.6a09e667f3bcdp-1")
LN2 = float.fromhex("0x1.62e42fefa39efp-1")
PIO2 = float.fromhex("0x1.921fb54442d18p+0")
TWO_M53 = 2.0 ** -53

# Philox4x64 constants from Salmon et al. (SC'11): round multipliers and the
# Weyl key increments (golden ratio and sqrt(3) - 1 in 0.64 fixed point).
_PHILOX_M0 = 0xD2E7470EE14C6C93
_PHILOX_M1 = 0xCA5A826395121157
_PHILOX_W0 = 0x9E3779B97F4A7C15
_PHILOX_W1 = 0xBB67AE8584CAA73B
_MASK64 = (1 << 64) - 1


def philox4x64_10_py(counter, key):
    """Philox4x64-10 of one 4x64-bit counter under a 2x64-bit key.

    Written from the SC'11 definition: ten rounds; each round multiplies words
    0 and 2 by the two multipliers (full 128-bit products), and the new block
    is (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0); the key is bumped by the Weyl
    constants before every round after the first.  Pure Python integers.
    """
    c0, c1, c2, c3 = (int(x) & _MASK64 for x in counter)
    k0, k1 = (int(x) & _MASK64 for x in key)
    for rnd in range(10):
        if rnd:
            k0 = (k0 + _PHILOX_W0) & _MASK64
            k1 = (k1 + _PHILOX_W1) & _MASK64
        p0 = _PHILOX_M0 * c0
        p1 = _PHILOX_M1 * c2
        hi0, lo0 = p0 >> 64, p0 & _MASK64
        hi1, lo1 = p1 >> 64, p1 & _MASK64
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return (c0, c1, c2, c3)


def philox_words(seed, domain, column, nblocks):
    """Words of counter blocks (q, column, 0, 0), q = 0 .. nblocks-1.

    numpy's Philox increments its 256-bit counter before producing a block,
    so starting one below (q = 0, column) yields exactly the blocks wanted.
    Returns a (nblocks, 4) uint64 array.
    """
    start = (int(column) << 64) - 1
    bg = np.random.Philox(key=(int(seed) & _MASK64) | (int(domain) << 64),
                          counter=start % (1 << 256))
    return bg.random_raw(4 * nblocks).reshape(nblocks, 4)


def _ln(u):
    """ln u for u in (0, 1], by the spec's frexp + atanh-series steps."""
    f, e = np.frexp(u)
    low = f < SQRT_HALF
    f = np.where(low, f * 2.0, f)
    e = np.where(low, e - 1, e).astype(np.float64)
    s = (f - 1.0) / (f + 1.0)
    z = s * s
    p = np.full_like(s, 1.0 / 21.0)
    for j in range(9, -1, -1):
        p = p * z + 1.0 / (2 * j + 1)
    return e * LN2 + (s + s) * p


def _cos_sin_2pi(u):
    """(cos 2 pi u, sin 2 pi u) for u in [0, 1), by quadrant + Taylor."""
    t = 4.0 * u
    q = np.floor(t)
    phi = (t - q) * PIO2
    x = phi * phi
    ps = np.ones_like(phi)
    pc = np.ones_like(phi)
    for k in range(11, 0, -1):
        ps = 1.0 - (x * ps) * (1.0 / ((2 * k) * (2 * k + 1)))
        pc = 1.0 - (x * pc) * (1.0 / ((2 * k - 1) * (2 * k)))
    sn = phi * ps
    cs = pc
    qi = q.astype(np.int64)
    cos_t = np.select([qi == 0, qi == 1, qi == 2], [cs, -sn, -cs], sn)
    sin_t = np.select([qi == 0, qi == 1, qi == 2], [sn, cs, -sn], -cs)
    return cos_t, sin_t


def _box_muller(wa, wb):
    """Two Gaussians from two 64-bit words (spec: uniforms, then Box--Muller)."""
    u1 = ((wa >> np.uint64(11)) + np.uint64(1)).astype(np.float64) * TWO_M53
    u2 = (wb >> np.uint64(11)).astype(np.float64) * TWO_M53
    r = np.sqrt(-2.0 * _ln(u1))
    c, s = _cos_sin_2pi(u2)
    return r * c, r * s


def normal_column(seed, n, column, domain=0):
    """Global sketch column ``column`` (length n) in float64."""
    nb = (n + 3) // 4
    w = philox_words(seed, domain, column, nb)
    z0, z1 = _box_muller(w[:, 0], w[:, 1])
    z2, z3 = _box_muller(w[:, 2], w[:, 3])
    out = np.empty(4 * nb, dtype=np.float64)
    out[0::4] = z0
    out[1::4] = z1
    out[2::4] = z2
    out[3::4] = z3
    return out[:n]


def normal_v1(seed, n, col0, ncols, dtype=np.float64, domain=0):
    """Sketch block: columns [col0, col0 + ncols) of the n x inf sketch.

    Returns an (n, ncols) Fortran-ordered array of ``dtype``; float32 values
    are the float64 values rounded to nearest-even.
    """
    out = np.empty((n, ncols), dtype=np.float64, order="F")
    for j in range(ncols):
        out[:, j] = normal_column(seed, n, col0 + j, domain)
    if np.dtype(dtype) == np.float32:
        return out.astype(np.float32, order="F")
    return out
