"""Brute-force checks that pin the oracle -- TEST INFRASTRUCTURE ONLY.

Pure Python (arbitrary-precision integers, exact rationals), written independently
of ``oracle.c`` and by different methods, so that a mistake in the oracle shows up
as a disagreement here:

* ``leaf``: the integer b-th root by a float candidate plus exact big-integer
  correction (the oracle bisects);
* ``stratified_targets``: the stratified target from its rational definition
  floor((k + u/2^64) * Q / B) (the oracle uses a 128-bit nested-floor form);
* ``linear_sample``: inverse CDF by a linear prefix scan (the oracle descends a
  binary tree);
* ``stack_from_stream``: frame stacks from the ingested stream itself (the oracle
  reads ring slots and checks episode/step metadata);
* ``nearest_f32`` / ``nearest_bf16``: correct rounding of an exact rational.
"""
from fractions import Fraction
import math
import struct


def frac_bits(a, b):
    """Fractional bits of the quantised leaf: floor(32(1 - a/b)), capped at 31."""
    return min(31, (32 * (b - a)) // b)


def leaf(p, a=3, b=5):
    """floor(2^F * p^(a/b)) for an integer priority p >= 0, exactly."""
    if p == 0:
        return 0
    F = frac_bits(a, b)
    target = (p ** a) << (b * F)  # q^b <= target < (q+1)^b
    q = int(round(float(target) ** (1.0 / b)))
    while q ** b > target:
        q -= 1
    while (q + 1) ** b <= target:
        q += 1
    return q


def stratified_targets(Q, B, uniforms):
    """t_k = floor((k + u_k / 2^64) * Q / B) as an exact rational floor."""
    return [((k << 64) + int(u)) * Q // (B << 64) for k, u in enumerate(uniforms)]


def linear_sample(leaves, t):
    """First slot whose inclusive prefix sum exceeds t (linear scan)."""
    acc = 0
    for i, q in enumerate(leaves):
        acc += int(q)
        if acc > t:
            return i
    raise ValueError("target beyond total priority")


def is_weights(leaves, size, idx, beta):
    """Schaul et al. importance weights, max-normalised over the batch, exact rationals
    for P(i) and the power taken in floating point."""
    Q = sum(int(q) for q in leaves)
    raw = [(size * Fraction(int(leaves[i]), Q)) ** 1 for i in idx]
    w = [float(x) ** (-beta) for x in raw]
    m = max(w)
    return [x / m for x in w]


def is_weights_buffer(leaves, size, idx, beta):
    """The same weights normalised by the largest weight any stored transition
    could receive: that of the smallest non-zero leaf of the buffer."""
    Q = sum(int(q) for q in leaves)
    qmin = min(int(q) for q in leaves if int(q) > 0)
    m = float(size * Fraction(qmin, Q)) ** (-beta)
    return [float(size * Fraction(int(leaves[i]), Q)) ** (-beta) / m for i in idx]


def stack_from_stream(stream_eps, stream_frames, capacity, total, pos, K):
    """Frame stack for the transition at stream position ``pos``.

    The stack holds the K observations at stream positions pos-K+1 .. pos, oldest
    first; a position that belongs to another episode, lies before the stream
    start, or has already been evicted from the ring (pos' < total - capacity) is
    all zeros.
    """
    out = []
    for k in range(K):
        p = pos - (K - 1 - k)
        ok = p >= 0 and p >= total - capacity and stream_eps[p] == stream_eps[pos]
        out.append(stream_frames[p] if ok else None)
    return out


def _f32_bits(x):
    return struct.unpack("<I", struct.pack("<f", x))[0]


def _f32_from_bits(u):
    return struct.unpack("<f", struct.pack("<I", u))[0]


def nearest_f32(q: Fraction):
    """The float32 nearest to the exact rational q (ties to even), for |q| in the
    normal range or zero."""
    if q == 0:
        return 0.0
    sign = -1 if q < 0 else 1
    a = abs(q)
    e = math.floor(math.log2(a.numerator) - math.log2(a.denominator))
    # fix e so that 2^e <= a < 2^(e+1)
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    scale = Fraction(2) ** (23 - e)
    m = a * scale  # in [2^23, 2^24)
    lo = math.floor(m)
    rem = m - lo
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and lo % 2 == 1):
        lo += 1
    return sign * float(Fraction(lo) / scale)


def nearest_bf16_bits(q: Fraction):
    """bfloat16 bit pattern nearest to the exact rational q (ties to even), normal
    range or zero."""
    if q == 0:
        return 0
    sign = 0x8000 if q < 0 else 0
    a = abs(q)
    e = 0
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    scale = Fraction(2) ** (7 - e)
    m = a * scale  # in [2^7, 2^8)
    lo = math.floor(m)
    rem = m - lo
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and lo % 2 == 1):
        lo += 1
    if lo == 256:
        lo = 128
        e += 1
    return sign | ((e + 127) << 7) | (lo - 128)
