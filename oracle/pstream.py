"""Oracle P stream — test infrastructure only (see ``oracle/__init__``).

The paper samples the projection from a per-layer seed, P ~ N(0, 1/r) with P of
shape n x r, and re-samples it with the same seed in the optimizer step
(Alg. 1 and Alg. 3, §3.3 "Random Projection Matrix").  It does not fix a
generator, so this oracle fixes one documented stream that the GPU library also
implements, independently, from the same definition:

* Philox4x32-10, the counter-based generator of Salmon, Moraes, Dror & Shaw,
  "Parallel Random Numbers: As Easy as 1, 2, 3" (SC'11): 10 rounds of the
  multiply-xor S-box with the published multipliers and Weyl key increments.
* Box-Muller (Box & Muller, 1958): a pair of uniforms (u, v) gives
  sqrt(-2 ln u) * (cos 2 pi v, sin 2 pi v).  The log, sine and cosine are a
  fixed sequence of IEEE fp32 add/sub/mul/div/sqrt operations (no fused
  multiply-add), written here in numpy float32 so that every operation rounds
  exactly as it does on the GPU.  The series are Taylor series (sin, cos) and
  the atanh series for log; their coefficients are the fp32 roundings of the
  exact rationals 1/k! and 1/k.

Element (i, j) of G (unscaled, N(0,1)):
    key     = (seed mod 2^32, seed >> 32)
    counter = (i >> 2, j, 0, 0)
    (w0, w1, w2, w3) = Philox4x32-10(counter, key)
    (a, b)  = (w0, w1) if (i & 2) == 0 else (w2, w3)
    radius from a (23-bit code), angle from b (24-bit code)
    G[i, j] = rho * cos(theta) if i is even else rho * sin(theta)

P = G / sqrt(r) (variance 1/r, the reading of §3.3 that makes P P^T ~ I).

The sparse Johnson-Lindenstrauss projection (the ablation's sparse JL
matrices, §5, after Dasgupta, Kumar and Sarlos, 2010; the paper fixes no
parameters) uses the same generator with counter word 2 set to a tag, s
signed unit draws per row and P = S / sqrt(s):
    draw q of row i, q = 0 .. s-1:
      (w0, w1, w2, w3) = Philox4x32-10((i, q >> 1, SJLT_TAG, 0), key)
      (a, b) = (w0, w1) for even q, (w2, w3) for odd q
      column floor(a r / 2^32), sign +1 if b < 2^31 else -1
    S[i, c] = sum of the signs of row i's draws that land on column c.
"""
from __future__ import annotations

import numpy as np

F32 = np.float32
U32 = np.uint32
U64 = np.uint64

# --------------------------------------------------------------------------
# Philox (SC'11).  A generic word-size implementation on Python integers,
# used for the 4x64 cross-check against numpy's Philox and for spot checks,
# and a vectorised 4x32 implementation for bulk generation.
# --------------------------------------------------------------------------

# Philox constants published with the generator: multipliers M0, M1 and the
# Weyl sequence increments (golden ratio and sqrt(3)-1 fractions).
PHILOX_CONSTANTS = {
    32: dict(M0=0xD2511F53, M1=0xCD9E8D57, W0=0x9E3779B9, W1=0xBB67AE85),
    64: dict(M0=0xD2E7470EE14C6C93, M1=0xCA5A826395121157,
             W0=0x9E3779B97F4A7C15, W1=0xBB67AE8584CAA73B),
}


def philox4_generic(counter, key, wordbits=32, rounds=10):
    """Philox4xW-R on Python ints.  counter: 4 words, key: 2 words."""
    c = PHILOX_CONSTANTS[wordbits]
    mask = (1 << wordbits) - 1
    x0, x1, x2, x3 = (int(v) & mask for v in counter)
    k0, k1 = (int(v) & mask for v in key)
    for rnd in range(rounds):
        if rnd > 0:  # key bump between rounds
            k0 = (k0 + c["W0"]) & mask
            k1 = (k1 + c["W1"]) & mask
        p0 = c["M0"] * x0
        p1 = c["M1"] * x2
        hi0, lo0 = p0 >> wordbits, p0 & mask
        hi1, lo1 = p1 >> wordbits, p1 & mask
        x0, x1, x2, x3 = hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0
    return (x0, x1, x2, x3)


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Vectorised Philox4x32-10.  All arguments broadcastable uint32 arrays.

    Products are formed in uint64 (32x32 -> 64 bits is exact)."""
    k = PHILOX_CONSTANTS[32]
    M0, M1 = U64(k["M0"]), U64(k["M1"])
    x0, x1, x2, x3 = (np.asarray(v, dtype=U64) & U64(0xFFFFFFFF) for v in (c0, c1, c2, c3))
    k0 = np.asarray(k0, dtype=U64) & U64(0xFFFFFFFF)
    k1 = np.asarray(k1, dtype=U64) & U64(0xFFFFFFFF)
    mask = U64(0xFFFFFFFF)
    for rnd in range(10):
        if rnd > 0:
            k0 = (k0 + U64(k["W0"])) & mask
            k1 = (k1 + U64(k["W1"])) & mask
        p0 = M0 * x0
        p1 = M1 * x2
        hi0, lo0 = p0 >> U64(32), p0 & mask
        hi1, lo1 = p1 >> U64(32), p1 & mask
        x0, x1, x2, x3 = hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0
    return tuple(v.astype(U32) for v in (x0, x1, x2, x3))


# --------------------------------------------------------------------------
# fp32 Box-Muller.  Every line below is one IEEE fp32 operation (numpy float32
# arithmetic rounds each +, -, *, /, sqrt to nearest-even and never fuses).
# --------------------------------------------------------------------------

def _c(num, den):
    """fp32 round-to-nearest of the rational num/den (both exact in fp32)."""
    return F32(num) / F32(den)


# atanh series for log: ln f = 2s (1 + s^2/3 + s^4/5 + s^6/7 + s^8/9), s=(f-1)/(f+1)
LOG_C3, LOG_C5, LOG_C7, LOG_C9 = _c(1, 3), _c(1, 5), _c(1, 7), _c(1, 9)
# Taylor series of sin and cos about 0 (signs folded into the coefficients)
SIN_C3, SIN_C5, SIN_C7, SIN_C9 = -_c(1, 6), _c(1, 120), -_c(1, 5040), _c(1, 362880)
COS_C2, COS_C4, COS_C6, COS_C8, COS_C10 = (-_c(1, 2), _c(1, 24), -_c(1, 720),
                                           _c(1, 40320), -_c(1, 3628800))
LN2_F32 = F32(np.log(np.float64(2.0)))          # fp32(ln 2)  = 0x3F317218
HALF_PI_F32 = F32(np.pi / 2.0)                  # fp32(pi/2)  = 0x3FC90FDB
SQRT2_MANT = 0x3504F3                           # mantissa bits of fp32(sqrt 2), just below sqrt 2


def log_f32(u):
    """ln(u) for fp32 u in (0, 1), as the fixed fp32 op sequence.

    u = 2^e * f with f in (sqrt(2)/2, sqrt(2)]; ln u = e ln2 + 2 atanh(s)."""
    u = np.asarray(u, dtype=F32)
    bits = u.view(U32)
    e = (bits >> U32(23)).astype(np.int32) - 127
    mant = bits & U32(0x7FFFFF)
    big = mant > U32(SQRT2_MANT)
    fbits = np.where(big, mant | U32(0x3F000000), mant | U32(0x3F800000)).astype(U32)
    e = e + big.astype(np.int32)
    f = fbits.view(F32)
    num = f - F32(1.0)
    den = f + F32(1.0)
    s = num / den
    s2 = s + s
    z = s * s
    p = LOG_C9
    p = p * z
    p = p + LOG_C7
    p = p * z
    p = p + LOG_C5
    p = p * z
    p = p + LOG_C3
    t = z * p
    t = s2 * t
    lnf = s2 + t
    el = e.astype(F32) * LN2_F32
    return el + lnf


def sin_f32(x):
    """sin(x) for fp32 x in [0, pi/4]: x + x*z*(c3 + z(c5 + z(c7 + z c9)))."""
    x = np.asarray(x, dtype=F32)
    z = x * x
    p = SIN_C9
    p = p * z
    p = p + SIN_C7
    p = p * z
    p = p + SIN_C5
    p = p * z
    p = p + SIN_C3
    xz = x * z
    t = xz * p
    return x + t


def cos_f32(x):
    """cos(x) for fp32 x in [0, pi/4]: 1 + z*(c2 + z(c4 + z(c6 + z(c8 + z c10))))."""
    x = np.asarray(x, dtype=F32)
    z = x * x
    q = COS_C10
    q = q * z
    q = q + COS_C8
    q = q * z
    q = q + COS_C6
    q = q * z
    q = q + COS_C4
    q = q * z
    q = q + COS_C2
    t = z * q
    return F32(1.0) + t


def radius_f32(a):
    """rho = sqrt(-2 ln u), u = (2*(a >> 9) + 1) * 2^-24, for 32-bit words a."""
    ka = np.asarray(a, dtype=U32) >> U32(9)
    u = (U32(2) * ka + U32(1)).astype(F32) * F32(2.0 ** -24)
    lnu = log_f32(u)
    t = lnu * F32(-2.0)
    return np.sqrt(t)


def angle_cs_f32(b):
    """(cos theta, sin theta), theta = 2 pi ((b >> 8) + 1/2) / 2^24, in fp32.

    Quadrant from the top two bits of the 24-bit code; within the quadrant the
    angle is reflected into [0, pi/4] with exact integer arithmetic."""
    kb = np.asarray(b, dtype=U32) >> U32(8)
    q = kb >> U32(22)
    c = kb & U32(0x3FFFFF)
    h = (c >> U32(21)) == U32(1)
    cr = np.where(h, U32(0x3FFFFF) - c, c).astype(U32)
    phi = (U32(2) * cr + U32(1)).astype(F32) * F32(2.0 ** -23)
    x = phi * HALF_PI_F32
    sx = sin_f32(x)
    cx = cos_f32(x)
    s_psi = np.where(h, cx, sx)
    c_psi = np.where(h, sx, cx)
    cos_t = np.select([q == 0, q == 1, q == 2, q == 3], [c_psi, -s_psi, -c_psi, s_psi])
    sin_t = np.select([q == 0, q == 1, q == 2, q == 3], [s_psi, c_psi, -s_psi, -c_psi])
    return cos_t.astype(F32), sin_t.astype(F32)


def box_muller_f32(a, b):
    """Two N(0,1) fp32 normals from two uint32 words: (rho cos, rho sin)."""
    rho = radius_f32(a)
    ct, st = angle_cs_f32(b)
    return rho * ct, rho * st


def seed_key(seed: int):
    seed = int(seed) & ((1 << 64) - 1)
    return U32(seed & 0xFFFFFFFF), U32(seed >> 32)


def gaussian_raw(seed: int, n: int, r: int) -> np.ndarray:
    """G (n x r, float32): the unscaled N(0,1) P stream for one layer seed."""
    if n <= 0 or r <= 0:
        return np.zeros((max(n, 0), max(r, 0)), dtype=F32)
    k0, k1 = seed_key(seed)
    nq = (n + 3) // 4
    p = np.arange(nq, dtype=U32)[:, None]
    j = np.arange(r, dtype=U32)[None, :]
    w0, w1, w2, w3 = philox4x32_10(p, j, U32(0), U32(0), k0, k1)
    g0, g1 = box_muller_f32(w0, w1)
    g2, g3 = box_muller_f32(w2, w3)
    out = np.empty((nq * 4, r), dtype=F32)
    out[0::4] = g0
    out[1::4] = g1
    out[2::4] = g2
    out[3::4] = g3
    return out[:n]


def gaussian_element(seed: int, i: int, j: int) -> np.float32:
    """One element of G, computed on its own (for sampled checks)."""
    k0, k1 = seed_key(seed)
    w = philox4x32_10(U32(i >> 2), U32(j), U32(0), U32(0), k0, k1)
    a, b = (w[0], w[1]) if (i & 2) == 0 else (w[2], w[3])
    g_even, g_odd = box_muller_f32(np.atleast_1d(a), np.atleast_1d(b))
    return (g_even if (i & 1) == 0 else g_odd)[0]


SJLT_TAG = 0x4A4C5350


def sparse_jl_raw(seed: int, n: int, r: int, s: int) -> np.ndarray:
    """S (n x r, float64 holding integers): the sparse JL stream, s draws per row."""
    if s < 1:
        raise ValueError("s >= 1 draws per row")
    k0, k1 = seed_key(seed)
    pairs = (s + 1) // 2
    i = np.arange(n, dtype=U32)[:, None]
    p = np.arange(pairs, dtype=U32)[None, :]
    w0, w1, w2, w3 = philox4x32_10(i, p, U32(SJLT_TAG), U32(0), k0, k1)
    # draw q = 2p takes (w0, w1) of pair p, draw q = 2p + 1 takes (w2, w3)
    a = np.stack([w0, w2], axis=-1).reshape(n, 2 * pairs)[:, :s]
    b = np.stack([w1, w3], axis=-1).reshape(n, 2 * pairs)[:, :s]
    col = ((a.astype(U64) * U64(r)) >> U64(32)).astype(np.int64)
    sign = np.where((b >> U32(31)) != 0, -1.0, 1.0)
    S = np.zeros((n, r), dtype=np.float64)
    np.add.at(S, (np.repeat(np.arange(n), s), col.ravel()), sign.ravel())
    return S


def projection(seed: int, n: int, r: int, identity: bool = False, sparse_s: int = 0) -> np.ndarray:
    """P in fp64: G / sqrt(r) (§3.3), the identity (requires r == n), or, with
    sparse_s = s > 0, the sparse JL projection S / sqrt(s)."""
    if identity:
        if r != n:
            raise ValueError("identity projection requires r == n")
        return np.eye(n, dtype=np.float64)
    if sparse_s:
        return sparse_jl_raw(seed, n, r, sparse_s) / np.sqrt(np.float64(sparse_s))
    return gaussian_raw(seed, n, r).astype(np.float64) / np.sqrt(np.float64(r))
