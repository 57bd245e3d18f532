"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: values the
paper prints (Table 1), hand derivations from its worked example, closed
forms (standard speculative sampling, Thm. 2, top-K verification), exact
enumeration of the output distribution (Thm. 1), the structural lemmas
(Lemmas 1-3), the T -> 0 degeneracy (Sec. 5.4), library routines (numpy's
Philox) and brute force.
"""

import json
import os
import zlib
from fractions import Fraction

import numpy as np
import pytest

from oracle import numerics, rheo
from oracle.drivers import enumerate_all, run_philox
from oracle.philox import philox4x64_10, draw_u64

GOLD = os.path.join(os.path.dirname(__file__), "golden")
F = Fraction


def _load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


# --------------------------------------------------------------------------
# Philox4x64-10
# --------------------------------------------------------------------------

def test_philox_known_answer():
    kat = _load("philox4x64_kat.json")
    ctr = [int(x, 16) for x in kat["counter"]]
    key = [int(x, 16) for x in kat["key"]]
    assert [hex(x) for x in philox4x64_10(ctr, key)] == kat["output"]


def test_philox_matches_numpy_bit_generator():
    # numpy.random.Philox is Philox4x64-10; it increments the counter before
    # producing a block, so counter c - 1 yields the block for c.
    rng = np.random.default_rng(1)
    for _ in range(20):
        ctr = [int(x) for x in rng.integers(0, 2 ** 63, 4, dtype=np.uint64)]
        key = [int(x) for x in rng.integers(0, 2 ** 63, 2, dtype=np.uint64)]
        c = sum(w << (64 * i) for i, w in enumerate(ctr))
        cm = (c - 1) % (1 << 256)
        ctr_m1 = [(cm >> (64 * i)) & ((1 << 64) - 1) for i in range(4)]
        bg = np.random.Philox(counter=ctr_m1, key=key)
        want = [int(x) for x in bg.random_raw(4)]
        assert list(philox4x64_10(ctr, key)) == want


# --------------------------------------------------------------------------
# canonical weights
# --------------------------------------------------------------------------

@pytest.mark.parametrize("T", [0.6, 1.0, 2.0, 0.8])
def test_canonical_weights_track_exp(T):
    rng = np.random.default_rng(7)
    d = -rng.uniform(0.0, 22.0 * T, 200000).astype(np.float32)
    w = numerics.canonical_weights(d, 0.0, T).astype(np.float64)
    exact = np.exp(d.astype(np.float64) / T) * 2.0 ** 30
    live = exact >= 1.0
    # fp32 rounding of t (3 ops, |t| <= 31) and the degree-6 polynomial give
    # < 5e-6 relative; truncation to an integer adds < 1 unit.
    err = np.abs(w[live] - exact[live])
    assert np.all(err <= 5e-6 * exact[live] + 1.0)
    assert np.all(w[exact < 2.0 ** -2] == 0)


def _f32_round(q):
    """Round-to-nearest-even fp32 of an exact rational (by comparison with
    the neighbours of a close guess; independent of numerics.fma32)."""
    g = np.float32(float(q))
    cands = [np.nextafter(g, np.float32(-np.inf)), g, np.nextafter(g, np.float32(np.inf))]
    def key(v):
        return (abs(F(float(v)) - q), int(np.array(v, np.float32).view(np.uint32)) & 1)
    return min(cands, key=key)


def test_fma32_is_correctly_rounded():
    # the canonical Horner steps are fused multiply-adds (one rounding); the
    # oracle's emulation must round a * b + c exactly once, including the
    # products that land near a midpoint of two fp32 values
    rng = np.random.default_rng(11)
    a = rng.uniform(-2 ** 20, 2 ** 20, 4000).astype(np.float32)
    b = rng.uniform(-0.5, 0.5, 4000).astype(np.float32)
    c = rng.uniform(-2 ** 30, 2 ** 30, 4000).astype(np.float32)
    # hard cases: c cancels most of a * b, and c = -(a * b rounded) + tiny
    ab32 = (a * b).astype(np.float32)
    c2 = (-ab32).astype(np.float32)
    c3 = (-ab32 + np.float32(2.0 ** -30)).astype(np.float32)
    A = np.concatenate([a, a, a])
    B = np.concatenate([b, b, b])
    C = np.concatenate([c, c2, c3])
    got = numerics.fma32(A, B, C)
    for x, y, z, g in zip(A[::7], B[::7], C[::7], got[::7]):
        want = _f32_round(F(float(x)) * F(float(y)) + F(float(z)))
        assert np.float32(g) == want, (x, y, z)
    # and it differs from the separately rounded product and sum somewhere
    sep = ((A * B).astype(np.float32) + C).astype(np.float32)
    assert np.any(sep != got)
    # a double-rounding trap: 4(1 + 2^-23) * 4(1 - 2^-23) + (2^28 + 32) lies
    # 2^-42 below the midpoint 2^28 + 48 of two fp32 values; rounded to fp64
    # first it becomes the midpoint, which then rounds to even (2^28 + 64)
    x = np.float32(4.0 * (1 + 2.0 ** -23))
    y = np.float32(4.0 - 2.0 ** -21)
    z = np.float32(2.0 ** 28 + 32)
    want = _f32_round(F(float(x)) * F(float(y)) + F(float(z)))
    assert want == np.float32(2.0 ** 28 + 32)
    assert np.float32(np.float64(x) * np.float64(y) + np.float64(z)) != want
    assert numerics.fma32(np.array([x]), np.array([y]), np.array([z]))[0] == want


def test_canonical_weight_edges():
    w = numerics.canonical_weights(np.array([0.0, -0.0, 5.0, -1e-30], np.float32), 0.0, 1.0)
    assert list(w) == [2 ** 30] * 4          # t clamped at 0: the reference weight
    assert numerics.canonical_weights(np.array([-40.0], np.float32), 0.0, 1.0)[0] == 0
    half = numerics.canonical_weights(np.array([-np.log(2.0)], np.float32), 0.0, 1.0)[0]
    assert abs(half - 2 ** 29) <= 2 ** 29 * 1e-6


# --------------------------------------------------------------------------
# Table 1 (printed values) and its hand-derived verification outcomes
# --------------------------------------------------------------------------

NAMES = {"A": 0, "B": 1, "C": 2}


def _table1_nd():
    return rheo.node_dist_from_weights([0, 1, 2], [5, 3, 2], m=1)


def test_table1_pool_rankings_and_survival():
    g = _load("table1.json")
    nd = _table1_nd()
    assert [float(F(w, nd.s1)) for w in nd.w1] == g["q"]
    assert {k: float(F(nd.tail.weight(NAMES[k]), nd.tail.total()))
            for k in ("B", "C")} == g["qtilde"]
    for row in g["rows"]:
        y = NAMES[row["Y"]]
        rule = row["proxy"]
        pool = rheo.make_pool(nd, g["K"], g["m"], y, proxy_rule=rule,
                              adhoc_proxy=g["adhoc_proxy"])
        sampled = [p for p in pool if p[2] == rheo.SAMPLED][0]
        want_proxy = g["rheo_proxy"] if rule == "rheo" else g["adhoc_proxy"]
        assert sampled[3] == want_proxy
        fills = [p for p in pool if p[2] == rheo.FILL]
        assert [p[1] for p in fills] == [NAMES[row["fill"]]]
        # the global ranking of the depth-1 tree = the pool ranking
        cfg = rheo.TreeConfig(K=3, m=1, depth=1, proxy_rule=rule,
                              adhoc_proxy=g["adhoc_proxy"])
        proc = rheo.build_tree(cfg, 1.0, lambda n, ns: _table1_nd())
        req = next(proc)
        try:
            proc.send(y)
        except StopIteration as stop:
            nodes = stop.value
        ranked = sorted(nodes[1:], key=rheo.priority)
        labels = ["Y" if n.kind == rheo.SAMPLED else "ABC"[n.token] for n in ranked]
        assert labels == row["ranking"]
        pt = rheo.prune(nodes, g["R"])
        surv = ["Y" if nodes[u].kind == rheo.SAMPLED else "ABC"[nodes[u].token]
                for u in pt.order[1:]]
        assert sorted(surv) == sorted(row["survivors"])


def _table1_factory(p, rule):
    cfg = rheo.TreeConfig(K=3, m=1, depth=1, proxy_rule=rule, adhoc_proxy=0.25)
    return lambda: rheo.rheo_step(cfg, 1.0, 2, lambda n, ns: _table1_nd(),
                                  lambda i: list(p))


@pytest.mark.parametrize("case", range(4))
def test_table1_derived_verification(case):
    g = _load("table1_derived.json")["cases"][case]
    res = enumerate_all(_table1_factory(g["p"], g["proxy"]))
    out = [F(0)] * 3
    acc = F(0)
    given = {}
    for prob, (nodes, pt, a, u) in res:
        tok = a[0] if a else u
        out[tok] += prob
        if a:
            acc += prob
        y = [n.token for n in nodes if n.kind == rheo.SAMPLED][0]
        given.setdefault(y, {}).setdefault(tok, F(0))
        given[y][tok] += prob
    assert out == [F(x) for x in g["output"]]
    assert acc == F(g["acceptance"])
    if "given_Y" in g:
        qt = {1: F(3, 5), 2: F(2, 5)}
        for yname, dist in g["given_Y"].items():
            y = NAMES[yname]
            got = {t: v / qt[y] for t, v in given[y].items() if v}
            assert got == {NAMES[k]: F(v) for k, v in dist.items()}


# --------------------------------------------------------------------------
# closed forms
# --------------------------------------------------------------------------

def _rand_weights(rng, V, lo=1, hi=1000):
    return [int(x) for x in rng.integers(lo, hi, V)]


def _first_token_stats(res):
    out, acc = {}, F(0)
    for prob, (nodes, pt, a, u) in res:
        tok = a[0] if a else u
        out[tok] = out.get(tok, F(0)) + prob
        if a:
            acc += prob
    return out, acc


@pytest.mark.parametrize("seed", range(6))
def test_standard_speculative_sampling_special_case(seed):
    # K = 1, m = 0: one sampled token with q~ = q; Algorithm 1 is standard
    # rejection sampling, acceptance = sum_x min(p(x), q(x)) (Sec. 2.2).
    rng = np.random.default_rng(seed)
    V = int(rng.integers(3, 7))
    q = _rand_weights(rng, V)
    p = _rand_weights(rng, V)
    cfg = rheo.TreeConfig(K=1, m=0, depth=1)
    fac = lambda: rheo.rheo_step(cfg, 1.0, 1,
                                 lambda n, ns: rheo.node_dist_from_weights(list(range(V)), q, m=0),
                                 lambda i: list(p))
    out, acc = _first_token_stats(enumerate_all(fac))
    qs, ps = F(sum(q)), F(sum(p))
    assert acc == sum(min(F(a) / ps, F(b) / qs) for a, b in zip(p, q))
    assert out == {v: F(p[v]) / ps for v in range(V)}


@pytest.mark.parametrize("seed", range(6))
def test_topk_verification_closed_form(seed):
    # s = -1 (sampled slot pruned): acceptance = sum over the candidates of p
    # (Thm. 2, last sentence).  K = 3, m = 2, R = 2 keeps x_1, x_2 only.
    rng = np.random.default_rng(100 + seed)
    V = int(rng.integers(4, 8))
    q = _rand_weights(rng, V)
    p = _rand_weights(rng, V)
    cfg = rheo.TreeConfig(K=3, m=2, depth=1)
    nd = rheo.node_dist_from_weights(list(range(V)), q, m=2)
    fac = lambda: rheo.rheo_step(cfg, 1.0, 2, lambda n, ns: nd, lambda i: list(p))
    out, acc = _first_token_stats(enumerate_all(fac))
    ps = F(sum(p))
    assert acc == (F(p[nd.support[0]]) + F(p[nd.support[1]])) / ps
    assert out == {v: F(p[v]) / ps for v in range(V)}


def _thm2(q, p, n, m):
    """eq. (rheo-acc) and its upper bound, from q, p (weights) and pool n."""
    V = len(q)
    qs, ps = F(sum(q)), F(sum(p))
    order = rheo.rank_order(list(range(V)), q)
    top = order[:n - 1]
    lead = order[:m]
    z = 1 - sum(F(q[v]) / qs for v in lead)
    qt = {v: (F(q[v]) / qs / z if v not in lead else F(0)) for v in range(V)}
    pp = {v: F(p[v]) / ps for v in range(V)}
    rnum = {v: max(F(0), pp[v] - qt[v]) for v in range(V)}
    rz = sum(rnum.values())
    xn = order[n - 1]
    r_xn = rnum[xn] / rz if rz else F(0)
    acc = (sum(pp[v] for v in top)
           + sum(min(pp[v], qt[v]) for v in range(V) if v not in top)
           + r_xn * sum(max(F(0), qt[v] - pp[v]) for v in top))
    topn = order[:n]
    bound = (sum(pp[v] for v in topn)
             + sum(min(pp[v], qt[v]) for v in range(V) if v not in topn))
    return acc, bound


@pytest.mark.parametrize("seed", range(10))
def test_thm2_single_layer_acceptance(seed):
    rng = np.random.default_rng(200 + seed)
    V = int(rng.integers(4, 9))
    n = int(rng.integers(2, min(V, 5)))
    m = int(rng.integers(0, n))
    q = _rand_weights(rng, V)
    p = _rand_weights(rng, V)
    nd = rheo.node_dist_from_weights(list(range(V)), q, m=m)
    cfg = rheo.TreeConfig(K=n, m=m, depth=1, eps=2.0 ** -40)
    fac = lambda: rheo.rheo_step(cfg, 1.0, n, lambda a, b: nd, lambda i: list(p))
    out, acc = _first_token_stats(enumerate_all(fac))
    want, bound = _thm2(q, p, n, m)
    assert acc == want
    assert acc <= bound
    ps = F(sum(p))
    assert out == {v: F(p[v]) / ps for v in range(V)}


def _rrsw(q, p, n, m):
    """eq. (rrsw-acc), App. D.2: the pool of Thm. 2 verified leads-first."""
    V = len(q)
    qs, ps = F(sum(q)), F(sum(p))
    order = rheo.rank_order(list(range(V)), q)
    top = order[:n - 1]
    lead = order[:m]
    z = 1 - sum(F(q[v]) / qs for v in lead)
    qt = {v: (F(q[v]) / qs / z if v not in lead else F(0)) for v in range(V)}
    pp = {v: F(p[v]) / ps for v in range(V)}
    A = sum(pp[v] for v in lead)
    pt = {v: (pp[v] / (1 - A) if v not in lead else F(0)) for v in range(V)}
    rnum = {v: max(F(0), pt[v] - qt[v]) for v in range(V)}
    rz = sum(rnum.values())
    xn = order[n - 1]
    r_xn = rnum[xn] / rz if rz else F(0)
    return (sum(pp[v] for v in top)
            + sum(min(pp[v], (1 - A) * qt[v]) for v in range(V) if v not in top)
            + (1 - A) * r_xn * sum(max(F(0), qt[v] - pt[v]) for v in top))


@pytest.mark.parametrize("seed", range(10))
def test_rrsw_single_layer_acceptance(seed):
    # App. D.2: the same pool verified leads-first (RRSw) accepts exactly
    # eq. (rrsw-acc) and stays lossless
    rng = np.random.default_rng(300 + seed)
    V = int(rng.integers(4, 9))
    n = int(rng.integers(2, min(V, 5)))
    m = int(rng.integers(1, n))
    q = _rand_weights(rng, V)
    p = _rand_weights(rng, V)
    nd = rheo.node_dist_from_weights(list(range(V)), q, m=m)
    cfg = rheo.TreeConfig(K=n, m=m, depth=1, verifier="rrsw")
    fac = lambda: rheo.rheo_step(cfg, 1.0, n, lambda a, b: nd, lambda i: list(p))
    out, acc = _first_token_stats(enumerate_all(fac))
    assert acc == _rrsw(q, p, n, m)
    ps = F(sum(p))
    assert out == {v: F(p[v]) / ps for v in range(V)}


@pytest.mark.parametrize("seed", range(4))
def test_rrsw_equals_rheo_without_leads(seed):
    # m = 0: no lead precedes the sampled child, so both verifiers take the
    # same decisions (eq. (rrsw-acc) reduces to eq. (rheo-acc) with A = 0)
    rng = np.random.default_rng(400 + seed)
    V = int(rng.integers(4, 8))
    n = int(rng.integers(2, min(V, 5)))
    q = _rand_weights(rng, V)
    p = _rand_weights(rng, V)
    nd = rheo.node_dist_from_weights(list(range(V)), q, m=0)
    res = {}
    for ver in ("rheo", "rrsw"):
        cfg = rheo.TreeConfig(K=n, m=0, depth=1, verifier=ver)
        fac = lambda: rheo.rheo_step(cfg, 1.0, n, lambda a, b: nd, lambda i: list(p))
        res[ver] = _first_token_stats(enumerate_all(fac))
    assert res["rheo"] == res["rrsw"]
    assert _rrsw(q, p, n, 0) == _thm2(q, p, n, 0)[0]


@pytest.mark.parametrize("seed", range(6))
def test_pure_topk_tree_acceptance(seed):
    # the pure top-K tree (Sec. 2.1, no sampled slot) verified by the same
    # sequential tests accepts sum_{Top_n} p and is lossless
    rng = np.random.default_rng(500 + seed)
    V = int(rng.integers(4, 8))
    n = int(rng.integers(1, V))
    q = _rand_weights(rng, V)
    p = _rand_weights(rng, V)
    nd = rheo.node_dist_from_weights(list(range(V)), q, m=1)
    cfg = rheo.TreeConfig(K=n, m=1, depth=1, mode="topk")
    fac = lambda: rheo.rheo_step(cfg, 1.0, n, lambda a, b: nd, lambda i: list(p))
    out, acc = _first_token_stats(enumerate_all(fac))
    ps = F(sum(p))
    assert acc == sum(F(p[v]) for v in nd.support[:n]) / ps
    assert out == {v: F(p[v]) / ps for v in range(V)}


# --------------------------------------------------------------------------
# Thm. 1: losslessness by exact enumeration over several steps
# --------------------------------------------------------------------------

def _logits_fn(seed, V, scale=2.0):
    """Deterministic random logits as a function of (role, prefix)."""
    cache = {}

    def f(role, prefix):
        k = (role, prefix)
        if k not in cache:
            ent = [seed, 1 if role == "d" else 2, len(prefix)] + [int(x) for x in prefix]
            rng = np.random.default_rng(ent)
            cache[k] = rng.normal(0, scale, V).astype(np.float32)
        return cache[k]
    return f


def _path(nodes, uid):
    out = []
    while uid > 0:
        out.append(nodes[uid].token)
        uid = nodes[uid].parent
    return tuple(reversed(out))


def _one_step(cfg, T, R, pre, lf, model, cache):
    """One step from prefix ``pre``: returns the emitted tokens."""
    def dd(node, nodes):
        k = ("d", pre + _path(nodes, node.uid))
        if k not in cache:
            cache[k] = rheo.node_dist_from_logits(
                lf(*k), cfg.m, T, cfg.support, cfg.construct_tempered, model,
                cfg.construct_full)
        return cache[k]
    holder = {}

    def tp(i):
        nodes, pt = holder["nodes"], holder["pt"]
        k = ("t", pre + _path(nodes, pt.order[i]))
        if k not in cache:
            w = rheo.target_weights(lf(*k), T, model)
            cache[k] = list(w) if model == "fp64" else [int(x) for x in w]
        return cache[k]

    nodes = yield from rheo.build_tree(cfg, T, dd)
    pt = rheo.prune(nodes, R)
    holder["nodes"], holder["pt"] = nodes, pt
    acc, u = yield from rheo.verify(nodes, pt, tp, cfg.verifier)
    return tuple(acc) + (u,)


def _multi_step_dist(cfg, T, R, L, lf, model):
    """Exact distribution of the first L emitted tokens over as many steps as
    needed (each step starts from the prefix the previous ones emitted)."""
    cache, memo = {}, {}

    def step_dist(pre):
        if pre not in memo:
            d = {}
            for prob, em in enumerate_all(lambda: _one_step(cfg, T, R, pre, lf, model, cache)):
                d[em] = d.get(em, F(0)) + prob
            memo[pre] = d
        return memo[pre]

    def first(pre, need):
        out = {}
        for em, prob in step_dist(pre).items():
            if len(em) >= need:
                key = em[:need]
                out[key] = out.get(key, F(0)) + prob
            else:
                for rest, p2 in first(pre + em, need - len(em)).items():
                    out[em + rest] = out.get(em + rest, F(0)) + prob * p2
        return out
    return first((), L)


def _target_seq_prob(seq, T, lf, model):
    prob = F(1)
    for t in range(len(seq)):
        row = lf("t", tuple(seq[:t]))
        P = rheo.target_weights(row, T, model)
        P = [F(x) for x in (P if model == "fp64" else [int(v) for v in P])]
        prob *= P[seq[t]] / sum(P)
    return prob


LOSSLESS_CASES = [
    # V, K, m, depth, R, T, support, tempered, model, L
    (5, 2, 1, 2, 3, 1.0, 0, False, "canonical", 2),
    (5, 3, 1, 2, 4, 0.5, 0, False, "canonical", 2),
    (4, 3, 0, 2, 5, 2.0, 0, False, "canonical", 2),
    (5, 3, 2, 1, 3, 1.0, 0, False, "canonical", 3),
    (6, 3, 1, 2, 2, 1.0, 4, False, "canonical", 2),
    (5, 2, 1, 2, 4, 0.5, 0, True, "canonical", 2),
    (4, 2, 1, 3, 6, 1.0, 0, False, "canonical", 2),
    (5, 3, 1, 2, 4, 1.0, 0, False, "fp64", 2),
    (5, 2, 0, 2, 3, 0.5, 3, False, "fp64", 2),
]
# every budget R from 1 to |U| on two small trees (Thm. 1 holds for all R)
LOSSLESS_CASES += [(4, 2, 1, 2, R, 1.0, 0, False, "canonical", 2) for R in range(1, 7)]
LOSSLESS_CASES += [(5, 3, 0, 2, R, 0.7, 0, False, "canonical", 2) for R in (1, 2, 5, 9)]
LOSSLESS_CASES += [
    (6, 4, 2, 2, 7, 1.0, 5, False, "canonical", 2),
    (6, 4, 3, 1, 4, 0.8, 0, True, "canonical", 2),
    (4, 2, 0, 3, 4, 2.0, 0, True, "fp64", 2),
    (5, 2, 1, 2, 3, 1.0, 0, False, "canonical", 3),
]


# the leads-first baseline (App. D.2) and the pure top-K tree are lossless too
LOSSLESS_CASES += [
    (5, 3, 1, 2, 4, 1.0, 0, False, "canonical", 2, "rrsw"),
    (5, 3, 2, 2, 5, 0.6, 0, False, "canonical", 2, "rrsw"),
    (6, 4, 2, 2, 6, 1.0, 5, False, "canonical", 2, "rrsw"),
    (4, 3, 1, 2, 3, 1.0, 0, False, "canonical", 2, "rrsw"),
    (5, 3, 1, 2, 5, 1.0, 0, False, "canonical", 2, "topk"),
    (5, 2, 1, 2, 2, 0.5, 0, False, "canonical", 2, "topk"),
]

# the whole-vocabulary construction reading of the sparse mode (Sec. 5.5):
# only the proxies change, so the output stays the target's
LOSSLESS_CASES += [
    (6, 3, 1, 2, 4, 1.0, 4, False, "canonical", 2, "rheo", True),
    (6, 3, 0, 2, 5, 0.6, 3, True, "canonical", 2, "rheo", True),
    (5, 3, 1, 2, 4, 1.0, 3, False, "canonical", 2, "rrsw", True),
]


@pytest.mark.parametrize("case", LOSSLESS_CASES)
def test_thm1_lossless_by_enumeration(case):
    V, K, m, D, R, T, S, tempered, model, L = case[:10]
    method = case[10] if len(case) > 10 else "rheo"
    full = case[11] if len(case) > 11 else False
    # a seed that does not depend on the interpreter's string hashing
    lf = _logits_fn(zlib.crc32(repr(case[:10]).encode()) & 0xFFFF, V)
    cfg = rheo.TreeConfig(K=K, m=m, depth=D, n_expand=min(K, 2), support=S,
                          construct_tempered=tempered, construct_full=full, model=model,
                          mode="topk" if method == "topk" else "rheo",
                          verifier="rrsw" if method == "rrsw" else "rheo")
    dist = _multi_step_dist(cfg, T, R, L, lf, model)
    assert sum(dist.values()) == 1
    for seq, prob in dist.items():
        want = _target_seq_prob(seq, T, lf, model)
        assert prob == want, (seq, float(prob), float(want))
        assert abs(float(prob) - float(want)) <= 1e-12
    # every sequence of positive target probability is reachable
    assert len(dist) == V ** L


def test_adhoc_proxy_breaks_losslessness():
    # Negative control (Sec. 4, Table 1): a proxy strictly between q(x_3) and
    # q(x_2) lets the sampled token's survival depend on its value (it
    # survives iff Y = x_2, whose fill is x_3), and the output drifts from p.
    V, L = 4, 1
    for seed in range(5):
        lf = _logits_fn(90 + seed, V)
        nd = rheo.node_dist_from_logits(lf("d", ()), 1, 1.0)
        q2, q3 = (float(F(w, nd.s1)) for w in nd.w1[1:3])
        proxy = 0.5 * (q2 + q3)
        cfg = rheo.TreeConfig(K=3, m=1, depth=1, proxy_rule="adhoc",
                              adhoc_proxy=proxy)
        dist = _multi_step_dist(cfg, 1.0, 2, L, lf, "canonical")
        assert sum(dist.values()) == 1
        assert any(dist.get((v,), F(0)) != _target_seq_prob((v,), 1.0, lf, "canonical")
                   for v in range(V))
        # the same instance with the Rheo proxy is lossless
        cfg = rheo.TreeConfig(K=3, m=1, depth=1)
        dist = _multi_step_dist(cfg, 1.0, 2, L, lf, "canonical")
        assert all(dist.get((v,), F(0)) == _target_seq_prob((v,), 1.0, lf, "canonical")
                   for v in range(V))


# --------------------------------------------------------------------------
# Lemmas 1-3 and normalisation on random trees
# --------------------------------------------------------------------------

def _random_tree(seed, V=60, K=5, m=1, D=4, T=1.0, S=0):
    lf = _logits_fn(seed, V, scale=2.5)
    cfg = rheo.TreeConfig(K=K, m=m, depth=D, n_expand=K, support=S)
    dd = lambda node, nodes: rheo.node_dist_from_logits(
        lf("d", _path(nodes, node.uid)), m, T, S)
    return run_philox(rheo.build_tree(cfg, T, dd), 0x1234 + seed, 0), cfg


@pytest.mark.parametrize("seed", range(5))
def test_lemmas_and_normalisation(seed):
    m = seed % 3
    nodes, cfg = _random_tree(seed, m=m, S=(40 if seed % 2 else 0))
    for n in nodes:
        if not n.expanded:
            continue
        nd = n.dist
        kids = [nodes[c] for c in n.children]
        y = [c for c in kids if c.kind == rheo.SAMPLED][0]
        assert y.slot == m + 1                                   # rank m+1
        qx = [F(w, nd.s1) for w in nd.w1]
        assert sum(qx) == 1 and sum(F(w, nd.tail.total()) for w in nd.tail.weights) == 1
        if m:
            assert F(y.proxy) >= 0 and y.proxy <= float(qx[m - 1])
        assert y.proxy >= float(qx[m])                           # Lemma 1
        for c in kids:
            assert c.proxy <= 1.0
            assert c.score <= n.score                            # Lemma 2
            if c.kind == rheo.FILL:
                assert c.proxy <= y.proxy
        assert y.qtrue == float(F(nd.tail.weight(y.token), nd.tail.total()))
    for R in (1, 5, 17, len(nodes) - 1):
        pt = rheo.prune(nodes, R)                                # asserts closure
        assert len(pt.order) == R + 1


@pytest.mark.parametrize("m", [0, 1, 2])
def test_lemma3_slot_determinism(m):
    # Trees that prune to the same T_k admit their (k+1)-th node in the same
    # slot (topological invariance); when that slot is deterministic T_{k+1}
    # is identical, when it is sampled its token is distributed as q~.
    V = 6
    lf = _logits_fn(5 + m, V)
    cfg = rheo.TreeConfig(K=3, m=m, depth=2, n_expand=2)
    dd = lambda node, nodes: rheo.node_dist_from_logits(
        lf("d", _path(nodes, node.uid)), m, 1.0)
    res = enumerate_all(lambda: rheo.build_tree(cfg, 1.0, dd))
    total = len(res[0][1]) - 1
    for k in range(1, total):
        groups = {}
        for prob, nodes in res:
            ranked = sorted(nodes[1:], key=rheo.priority)
            tk = tuple((n.path, n.token) for n in ranked[:k])
            groups.setdefault(tk, []).append((prob, ranked[k], nodes))
        for tk, members in groups.items():
            slots = {m[1].path for m in members}
            assert len(slots) == 1
            kinds = {m[1].kind for m in members}
            assert len(kinds) == 1
            if kinds == {rheo.SAMPLED}:
                mass = sum(p for p, _, _ in members)
                by_tok = {}
                for p, n, nodes in members:
                    by_tok[n.token] = by_tok.get(n.token, F(0)) + p
                parent = members[0][2][members[0][1].parent]
                tail = parent.dist.tail
                for tok, p in by_tok.items():
                    assert p / mass == F(tail.weight(tok), tail.total())
            else:
                assert len({m[1].token for m in members}) == 1


# --------------------------------------------------------------------------
# T -> 0 degeneracy (Sec. 5.4)
# --------------------------------------------------------------------------

def test_low_temperature_degeneracy():
    V, K, D = 40, 4, 3
    single = []
    for seed in range(11, 17):
        lf = _logits_fn(seed, V, scale=3.0)
        cfg = rheo.TreeConfig(K=K, m=0, depth=D, mode="topk")
        dd = lambda node, nodes: rheo.node_dist_from_logits(
            lf("d", _path(nodes, node.uid)), 0, 1e-4)
        topk = run_philox(rheo.build_tree(cfg, 1e-4, dd), 77, 0)
        ref = [(n.token, n.parent, n.slot) for n in topk]
        for key in range(2):
            for m in (0, 1):
                cfg = rheo.TreeConfig(K=K, m=m, depth=D, eps=2.0 ** -80)
                dd = lambda node, nodes, m=m: rheo.node_dist_from_logits(
                    lf("d", _path(nodes, node.uid)), m, 1e-4)
                nodes = run_philox(rheo.build_tree(cfg, 1e-4, dd), 1000 + key, 0)
                # sampling degeneracy: Y is x_{m+1} whatever the draw
                for n in nodes:
                    if n.expanded:
                        y = [nodes[c] for c in n.children if nodes[c].kind == rheo.SAMPLED][0]
                        assert y.token == n.dist.support[m]
                sig = [(n.token, n.parent, n.slot) for n in nodes]
                if m == 0:
                    # dual degeneracy: the tree is the pure top-K tree
                    assert sig == ref
                else:
                    single.append(sig != ref)
    # single degeneracy for m = 1: the proxy min{q(x1), z} != q(x2) moves
    # the topology away from top-K on some instances
    assert any(single)


# --------------------------------------------------------------------------
# sampler
# --------------------------------------------------------------------------

def test_inverse_cdf_matches_linear_scan():
    rng = np.random.default_rng(3)
    P = rng.integers(0, 2 ** 30, 500).astype(np.int64)
    over = {int(v): int(rng.integers(0, 2 ** 60)) for v in rng.choice(500, 40, replace=False)}
    r = rheo.ResidualDist(P, 12345, over)
    w = [r.weight(v) for v in range(500)]
    assert r.total() == sum(w)
    for _ in range(200):
        t = int(rng.integers(0, 2 ** 62)) % r.total()
        acc, want = 0, None
        for v, x in enumerate(w):
            acc += x
            if acc > t:
                want = v
                break
        assert r.pick(t) == want


def test_philox_sampler_frequencies():
    from oracle.drivers import resolve_philox
    ids = [3, 7, 11, 20]
    wts = [5, 1, 3, 11]
    d = rheo.ExplicitDist(ids, wts)
    n = 40000
    counts = {i: 0 for i in ids}
    for j in range(n):
        counts[resolve_philox(rheo.Cat(1, j, d), 0xABCDEF, 0)] += 1
    tot = sum(wts)
    chi2 = sum((counts[i] - n * w / tot) ** 2 / (n * w / tot) for i, w in zip(ids, wts))
    assert chi2 < 16.3   # 3 d.o.f., p = 0.001


def test_harness_applies_the_method():
    # the workload's method reaches the oracle step: under RRSw a lead's test
    # (draw index 32 * level + its slot) comes before the sampled child's
    # (index 32 * level) at some layer; under Algorithm 1 never
    import synth
    from oracle.harness import oracle_step
    w = synth.WORKLOADS["tiny"]
    seen = {"rheo": False, "rrsw": False}
    for method in seen:
        for step in range(12):
            tr = []
            oracle_step(w.with_(method=method), 0, step, trace=tr)
            tests = [t[2] for t in tr if t[0] == "Bern"]
            for i, idx in enumerate(tests):
                if idx % 32 == 0 and any(j // 32 == idx // 32 for j in tests[:i]):
                    seen[method] = True
    assert seen == {"rheo": False, "rrsw": True}


@pytest.mark.parametrize("seed", range(4))
def test_whole_vocabulary_construction(seed):
    # Sec. 5.5 reading: construction over all of V, sampling on the top S.
    rng = np.random.default_rng(700 + seed)
    V, S, m, T = 40, 8, 1, 0.8
    l = (rng.normal(0, 2.0, V)).astype(np.float32)
    sparse = rheo.node_dist_from_logits(l, m, T, S)
    full = rheo.node_dist_from_logits(l, m, T, S, construct_full=True)
    dense = rheo.node_dist_from_logits(l, m, T, 0)
    # the support, its weights, order and tail are those of the sparse node
    assert full.support == sparse.support and full.w1 == sparse.w1
    assert full.tail.ids == sparse.tail.ids and full.tail.weights == sparse.tail.weights
    # the total is the dense node's, so q(x_i) are whole-vocabulary probabilities
    assert full.s1 == dense.s1 and full.support == dense.support[:S]
    assert full.w1 == dense.w1[:S]
    ex = np.exp(l.astype(np.float64) - l.max())
    for i, v in enumerate(full.support):
        q = full.w1[i] / full.s1
        assert abs(q - ex[v] / ex.sum()) <= 1e-6
    # at S = V the two readings coincide
    a = rheo.node_dist_from_logits(l, m, T, V, construct_full=True)
    b = rheo.node_dist_from_logits(l, m, T, V)
    assert a.s1 == b.s1 and a.w1 == b.w1


@pytest.mark.parametrize("seed", range(3))
def test_tree_mask(seed):
    # the mask the target forward needs (Sec. 2.1): ancestors by the node
    # records' own parent links, rows nested along the tree, lower triangular
    rng = np.random.default_rng(900 + seed)
    V, K, m, D, R = 12, 4, 1, 3, 14
    cfg = rheo.TreeConfig(K=K, m=m, depth=D, n_expand=2)
    dists = {}

    def dd(node, nodes):
        if node.uid not in dists:
            l = rng.normal(0, 2.0, V).astype(np.float32)
            dists[node.uid] = rheo.node_dist_from_logits(l, m, 1.0)
        return dists[node.uid]
    nodes = run_philox(rheo.build_tree(cfg, 1.0, dd), 0x1234 + seed, 0)
    pt = rheo.prune(nodes, R)
    mask, depth = rheo.tree_mask(nodes, pt)
    n = len(pt.order)
    pos = {u: i for i, u in enumerate(pt.order)}
    for i in range(n):
        anc = set()
        u = pt.order[i]
        while u != -1:
            anc.add(pos[u])
            u = nodes[u].parent
        assert {j for j in range(n) if mask[i][j]} == anc
        assert sum(mask[i]) == depth[i] + 1
        assert all(mask[i][j] == 0 for j in range(i + 1, n))
        if i:
            p = pt.parent[i]
            assert [mask[i][j] - mask[p][j] for j in range(n)] == [int(j == i) for j in range(n)]
