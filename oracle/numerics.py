"""Number models of the oracle.  TEST INFRASTRUCTURE ONLY.

The paper fixes no precision (it reports none).  Every decision the method
takes -- which token is sampled (Y ~ q~, Sec. 3.2; u* ~ r, Algorithm 1) and
whether a test ``eta <= ...`` passes (Algorithm 1) -- is a floating-point
comparison that turns into an integer.  So that two independent
implementations take identical decisions, each probability is represented by
an integer weight and every decision is an exact integer comparison
(reading stated in the design notes):

canonical model ("the kernel's precision")
    weight(l; ref, T) = floor(2**30 * 2**t) with t = fl32(fl32(l - ref) * kT),
    kT = fl32(log2(e) / T); 2**t is evaluated as 2**n * P(f) with n = rint(t),
    f = t - n in [-1/2, 1/2] (exact) and P the degree-6 Taylor polynomial of
    2**f in Horner form, each step p <- fl32(p * f + c_k) one fused
    multiply-add (a single rounding, IEEE 754 fusedMultiplyAdd), coefficients
    c_k = fp32((ln 2)^k / k! * 2**30) correctly rounded.  t is clamped to <= 0; t < -31 gives weight 0.  The
    integer result is (uint32)(P * 2**30) >> (-n), i.e. floor(P * 2**(30+n)).
    Weights are <= 2**30; sums over <= 262143 tokens fit in 48 bits.

fp64 model
    weight = exp((l - ref) / T) in fp64, used as an exact rational.  It is
    used only by the theory pins; the canonical model is checked against it
    within the quantisation bound.
"""

from decimal import Decimal, getcontext
from fractions import Fraction
import math

import numpy as np

WSHIFT = 30
LOG2E = 1.4426950408889634        # log2(e), the nearest double
T_CLAMP = -31.0                   # below this 2**(30+t) < 1/2: weight 0


def _poly_coeffs():
    """c_k = (ln 2)^k / k! * 2**30, k = 0..6, rounded to nearest fp32.
    Computed in 60-digit decimal arithmetic so the fp32 rounding is exact."""
    getcontext().prec = 60
    ln2 = Decimal(2).ln()
    out = []
    fact = Decimal(1)
    for k in range(7):
        if k:
            fact *= k
        exact = ln2 ** k / fact * (Decimal(2) ** WSHIFT)
        near = np.float32(float(exact))
        cands = [np.nextafter(near, np.float32(-np.inf)), near,
                 np.nextafter(near, np.float32(np.inf))]
        out.append(min(cands, key=lambda v: abs(Decimal(float(v)) - exact)))
    return [np.float32(c) for c in out]


POLY = _poly_coeffs()


def fma32(a, b, c):
    """Correctly rounded fp32 fused multiply-add a * b + c of fp32 arrays.
    The product is exact in fp64 (48 significant bits); the sum is rounded
    to odd in fp64 (rounded to nearest, its exact error from TwoSum (Knuth),
    and the odd one of the two fp64 neighbours of the exact sum when that
    error is not 0); rounding that to nearest fp32 gives the correctly
    rounded sum, since fp64 carries more than two bits beyond fp32 (Boldo
    and Melquiond, "Emulation of FMA and correctly rounded sums: proved
    algorithms using rounding to odd", IEEE Trans. Computers 57(4), 2008)."""
    x = np.asarray(a, dtype=np.float32).astype(np.float64) * np.asarray(b, np.float32).astype(np.float64)
    y = np.asarray(c, dtype=np.float32).astype(np.float64)
    x, y = np.broadcast_arrays(x, y)
    s = x + y
    bp = s - x
    e = (x - (s - bp)) + (y - bp)
    even = (s.view(np.uint64) & np.uint64(1)) == 0
    step = np.nextafter(s, np.where(e > 0, np.inf, -np.inf))
    s = np.where((e != 0) & even, step, s)
    return s.astype(np.float32)


def k_of_T(T):
    """kT = fp32(log2(e) / T) with T taken as an fp32 value (the ABI's type)."""
    return np.float32(LOG2E / float(np.float32(T)))


def canonical_weights(logits, ref, T):
    """Canonical integer weights of ``logits`` (an fp32 array) relative to the
    reference logit ``ref`` at temperature ``T``; returns an int64 array.

    This is the probability numerator of softmax(l / T) over the support:
    p(v) = weight(v) / sum(weights).  Every step is one fp32 operation."""
    l = np.asarray(logits, dtype=np.float32)
    d = (l - np.float32(ref)).astype(np.float32)
    t = (d * k_of_T(T)).astype(np.float32)
    t = np.minimum(t, np.float32(0.0))
    zero = t < np.float32(T_CLAMP)
    t = np.where(zero, np.float32(0.0), t).astype(np.float32)
    n = np.rint(t).astype(np.float32)
    f = (t - n).astype(np.float32)
    p = np.full(f.shape, POLY[6], dtype=np.float32)
    for c in POLY[5::-1]:
        p = fma32(p, f, c)
    u = p.astype(np.uint32)
    sh = (-n).astype(np.int64).astype(np.uint32)
    w = (u >> sh).astype(np.int64)
    w[zero] = 0
    return w


def fp64_weights(logits, ref, T):
    """fp64 model: exact rationals of exp((l - ref) / T) evaluated in fp64."""
    out = []
    for v in np.asarray(logits, dtype=np.float64):
        out.append(Fraction(math.exp((float(v) - float(ref)) / float(T))))
    return out
