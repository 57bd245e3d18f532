"""Drivers that resolve the random-choice requests of ``rheo.py``.
TEST INFRASTRUCTURE ONLY (see the package docstring).

run_philox     resolves every request with a Philox4x64-10 draw
               (counter layout in ``philox.py``):
                 Bern(num, den): eta = (U + 1) / 2**32 with U the 32-bit
                   draw, accept iff (U + 1) * den <= 2**32 * num  -- exact;
                   eta is in (0, 1], so a zero-probability candidate is never
                   accepted and a probability-one test always passes.
                 Cat(dist): t = floor(U64 * total / 2**64), the token is the
                   smallest id whose inclusive prefix weight exceeds t
                   (inverse CDF in token-id order).
enumerate_all  explores every outcome of every request with its exact
               probability (Fractions): Bern branches with min(1, num/den),
               Cat branches with weight/total.  The process is replayed from
               the start for each branch, which keeps the method code free
               of any bookkeeping for the enumeration.
"""

from fractions import Fraction

from .philox import draw_u64
from .rheo import Bern, Cat


def resolve_philox(req, rng_key, seq):
    """One request resolved by its Philox draw."""
    word = draw_u64(rng_key, req.purpose, seq, req.index)
    if isinstance(req, Bern):
        u = word >> 32
        return (u + 1) * int(req.den) <= (int(req.num) << 32)
    total = int(req.dist.total())
    t = (word * total) >> 64
    return req.dist.pick(t)


def run_philox(process, rng_key, seq, trace=None):
    """Run a request-yielding generator to completion under Philox draws.
    ``trace`` (a list) receives (request kind, purpose, index, outcome)."""
    try:
        req = next(process)
        while True:
            out = resolve_philox(req, rng_key, seq)
            if trace is not None:
                trace.append((type(req).__name__, req.purpose, req.index, out))
            req = process.send(out)
    except StopIteration as stop:
        return stop.value


def _branches(req):
    if isinstance(req, Bern):
        num, den = Fraction(req.num), Fraction(req.den)
        p = Fraction(1) if den == 0 or num >= den else num / den
        out = []
        if p > 0:
            out.append((True, p))
        if p < 1:
            out.append((False, 1 - p))
        return out
    total = Fraction(req.dist.total())
    return [(v, Fraction(w) / total) for v, w in req.dist.outcomes()]


def enumerate_all(factory):
    """Every complete outcome of ``factory()`` with its exact probability:
    a list of (probability, return value)."""
    results = []
    stack = [((), Fraction(1))]
    while stack:
        forced, prob = stack.pop()
        proc = factory()
        try:
            req = next(proc)
            i = 0
            while True:
                if i < len(forced):
                    req = proc.send(forced[i])
                    i += 1
                    continue
                for out, p in _branches(req):
                    stack.append((forced + (out,), prob * p))
                break
        except StopIteration as stop:
            results.append((prob, stop.value))
    return results
