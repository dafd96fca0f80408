"""Oracle: per-device variation factors and the device characteristic table
(Sec. V-A, generator step 2; Sec. IV-B).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The generator samples "the variation profile" to give every synaptic element
of every crossbar instance its own variation factor VF, and converts weights
to conductances through the device characteristic, "either using equations or
lookup tables" (Sec. V-A).  Sec. IV-B studies variations with sigma/mu = 10 %.
Readings (the figure that defines both is not in the text):

* ``G = G_nominal * VF`` for every device, padded positions included (they
  are physical devices).  VF is either supplied per device by the caller, or
  drawn as ``VF = max(0, 1 + sigma z)`` with z standard normal.
* z comes from a counter-based generator so that every device's factor is a
  pure function of (seed, device index): Philox-4x64 with 10 rounds (Salmon,
  Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3",
  SC 2011), counter ``(d, 0, 0, 0)`` for device index d, key ``(seed, 0)``;
  words x0, x1 of the output give ``u1 = ((x0 >> 11) + 1) 2^-53`` in (0, 1]
  and ``u2 = (x1 >> 11) 2^-53`` in [0, 1); Box-Muller
  ``z = sqrt(-2 ln u1) cos(2 pi u2)``.
* Device index ``d = a_glob (M N) + i N + j`` with the layer's array index
  ``a_glob = (c R + r) A + a`` (tile column c, tile row r, array a).
* The characteristic table f holds n >= 2 samples of the normalised
  conductance ``(G - g_min) / (g_max - g_min)`` at levels ``u = k / (n - 1)``;
  between samples it is linear.  The level is ``min(|w| / w_max, 1)`` for a
  continuous device and ``d / (2^b - 1)`` for a b-bit slice digit d.

Parity status: Philox is pinned bit for bit against numpy's independent
Philox-4x64 implementation; the normal draws by their moments; the table by
its samples, by linearity between them and by the identity table reproducing
the linear device; VF = 1 reproduces the unvaried mapping.
"""

from __future__ import annotations

import math

import numpy as np

M0 = 0xD2E7470EE14C6C93
M1 = 0xCA5A826395121157
W0 = 0x9E3779B97F4A7C15
W1 = 0xBB67AE8584CAA73B
MASK = (1 << 64) - 1


def philox4x64(counter, key, rounds=10):
    """One Philox-4x64 block: ``counter`` 4 ints, ``key`` 2 ints (Python
    integers, 64-bit arithmetic written out)."""
    c0, c1, c2, c3 = (int(v) & MASK for v in counter)
    k0, k1 = (int(v) & MASK for v in key)
    for rnd in range(rounds):
        if rnd:
            k0 = (k0 + W0) & MASK
            k1 = (k1 + W1) & MASK
        p0 = M0 * c0
        p1 = M1 * c2
        hi0, lo0 = p0 >> 64, p0 & MASK
        hi1, lo1 = p1 >> 64, p1 & MASK
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3


def _mul64(a, b):
    """Elementwise 64 x 64 -> (hi, lo) 64-bit products of uint64 arrays,
    through 32-bit halves."""
    m32 = np.uint64(0xFFFFFFFF)
    s32 = np.uint64(32)
    a_lo, a_hi = a & m32, a >> s32
    b_lo, b_hi = b & m32, b >> s32
    ll = a_lo * b_lo
    lh = a_lo * b_hi
    hl = a_hi * b_lo
    hh = a_hi * b_hi
    mid = (ll >> s32) + (lh & m32) + (hl & m32)
    lo = (ll & m32) | ((mid & m32) << s32)
    hi = hh + (lh >> s32) + (hl >> s32) + (mid >> s32)
    return hi, lo


def philox4x64_array(d, seed, rounds=10):
    """Philox-4x64 of counters ``(d, 0, 0, 0)`` (uint64 array d) under key
    ``(seed, 0)``: the four output words, each an array like d."""
    with np.errstate(over="ignore"):
        c0 = np.asarray(d, dtype=np.uint64).copy()
        c1 = np.zeros_like(c0)
        c2 = np.zeros_like(c0)
        c3 = np.zeros_like(c0)
        k0 = np.uint64(int(seed) & MASK)
        k1 = np.uint64(0)
        m0, m1 = np.uint64(M0), np.uint64(M1)
        for rnd in range(rounds):
            if rnd:
                k0 = np.uint64((int(k0) + W0) & MASK)
                k1 = np.uint64((int(k1) + W1) & MASK)
            hi0, lo0 = _mul64(np.full_like(c0, m0), c0)
            hi1, lo1 = _mul64(np.full_like(c2, m1), c2)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3


def normal_from_words(x0, x1):
    """Box-Muller on two 64-bit words per draw (fp64)."""
    u1 = ((np.asarray(x0, dtype=np.uint64) >> np.uint64(11)).astype(np.float64) + 1.0) * 2.0 ** -53
    u2 = (np.asarray(x1, dtype=np.uint64) >> np.uint64(11)).astype(np.float64) * 2.0 ** -53
    return np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * math.pi * u2)


def generated_factors(d, seed, sigma):
    """VF = max(0, 1 + sigma z) for device indices d."""
    x0, x1, _, _ = philox4x64_array(d, seed)
    return np.maximum(0.0, 1.0 + float(sigma) * normal_from_words(x0, x1))


def device_indices(a_glob0, A, M, N):
    """[A, M, N] device indices of the arrays a_glob0 .. a_glob0 + A - 1."""
    a = np.arange(A, dtype=np.uint64)[:, None, None] + np.uint64(a_glob0)
    i = np.arange(M, dtype=np.uint64)[None, :, None]
    j = np.arange(N, dtype=np.uint64)[None, None, :]
    return a * np.uint64(M * N) + i * np.uint64(N) + j


def characteristic(u, table):
    """Normalised conductance of level(s) u in [0, 1]: linear interpolation
    of ``table`` (n samples at k / (n - 1)); ``table`` None: the linear
    device, f(u) = u."""
    u = np.asarray(u, dtype=np.float64)
    if table is None:
        return u
    f = np.asarray(table, dtype=np.float64)
    n = f.size
    pos = np.clip(u, 0.0, 1.0) * (n - 1)
    k = np.minimum(np.floor(pos).astype(np.int64), n - 2)
    t = pos - k
    return f[k] + t * (f[k + 1] - f[k])
