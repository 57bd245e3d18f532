"""The RheoSampling hot path, step by step, in the paper's order.
TEST INFRASTRUCTURE ONLY (see the package docstring).

One *step* for one sequence is

  1. expand-then-rerank for D levels (Sec. 2.1): each selected parent gets a
     candidate pool of K slots -- the top-m tokens, one token Y sampled from
     the tail distribution q~, then the highest-ranked remaining tokens
     (Sec. 3.2, "Hybrid sampling mechanism"; App. C.1 "Hybrid candidate
     pool").  Y carries the proxy probability min{q(x_m), z} for
     construction and its true probability q~(Y) for verification (Sec. 3.2,
     "Dual treatment"; App. C.1 proxy list).  Path score = product of the
     proxies along the root-to-node path (App. C.1).  The next level expands
     the n_expand new nodes with the highest path scores (Sec. 2.1; App.
     C.4, step 1, where the K best-scoring nodes are the ones expanded).
  2. global top-R pruning by path score, ties broken by depth (shallower
     first) and then left-to-right sibling order (App. C.1, "Tie-breaking
     rule"), which keeps the pruned tree ancestor-closed.
  3. RheoVerification (Algorithm 1) applied layer by layer from the root
     (Thm. 1): accept the sampled child with probability min(1, p/q~);
     otherwise run sequential rejection over the remaining children under
     r = norm(max(0, p - q~)) (or r = p when the sampled child was pruned);
     if every child is rejected, emit u* ~ r.  At a leaf the algorithm has no
     candidates and reduces to u* ~ p.

Construction uses the untempered draft probabilities; sampling and
verification use temperature T (Sec. 5.4, "Decoupling tree construction from
temperature").  In sparse mode the draft logits are truncated to their top-S
entries before the softmax, and verification uses the same truncated q
(Sec. 3.2, "Efficient implementation via sparse distributions").

Random choices are *requests* yielded by generator functions:
  Cat(purpose, index, dist)   -> the driver sends back a token id
  Bern(purpose, index, num, den) -> the driver sends back True iff
                                     eta <= num / den for eta ~ U(0, 1]
so one implementation serves both the Philox driver and exact enumeration.
"""

import bisect
from dataclasses import dataclass, field
import itertools
from fractions import Fraction

import numpy as np

from . import numerics
from .philox import DRAFT, VERIFY, FINAL

LEAD, SAMPLED, FILL = 0, 1, 2
KIND_NAMES = {LEAD: "lead", SAMPLED: "sampled", FILL: "fill"}


# ---------------------------------------------------------------------------
# random-choice requests and the distributions they sample from
# ---------------------------------------------------------------------------

@dataclass
class Cat:
    """Sample one token from ``dist`` (an ExplicitDist or ResidualDist)."""
    purpose: int
    index: int
    dist: object


@dataclass
class Bern:
    """Accept iff eta <= num / den, eta ~ U(0, 1] (a ratio >= 1 always
    accepts, a zero numerator never does)."""
    purpose: int
    index: int
    num: object
    den: object


class ExplicitDist:
    """Integer (or rational) weights on a list of token ids.  Sampling is by
    inverse CDF over the ids in ascending order, or, with ``ranked``, over
    the ids in the order given (a sparse node's tail in rank order)."""

    def __init__(self, ids, weights, ranked=False):
        ids_np = np.asarray(ids, dtype=np.int64)
        order = (np.arange(len(ids_np)) if ranked
                 else np.argsort(ids_np, kind="stable"))
        self.ids = ids_np[order].tolist()
        if isinstance(weights, np.ndarray) and weights.dtype.kind in "iu":
            self.weights = weights[order].tolist()         # exact Python ints
        else:
            self.weights = [weights[i] for i in order]
        self._total = sum(self.weights)
        self._index = {v: i for i, v in enumerate(self.ids)}
        self._cum = None

    def total(self):
        return self._total

    def weight(self, v):
        i = self._index.get(int(v))
        return 0 if i is None else self.weights[i]

    def outcomes(self):
        return [(i, w) for i, w in zip(self.ids, self.weights) if w > 0]

    def pick(self, t):
        """First id, in this distribution's order, whose inclusive prefix
        weight exceeds ``t``."""
        if self._cum is None:
            self._cum = list(itertools.accumulate(self.weights))
        k = bisect.bisect_right(self._cum, t)
        if k >= len(self.ids):
            raise AssertionError("target beyond the total weight")
        return self.ids[k]


def _num(x):
    """Exact value of a weight: numpy integers become Python ints so that
    products never overflow; ints and Fractions pass through."""
    return int(x) if isinstance(x, np.integer) else x


class ResidualDist:
    """r over the whole vocabulary: weight(v) = F * P[v] except for the
    tokens listed in ``override`` (the tail support of q~ and the rejected
    candidates), which carry their own weight.  With F = 1 and only zeroed
    candidates overridden this is p with rejected candidates removed."""

    def __init__(self, P, F, override):
        self.P = P
        self.F = F
        self.override = dict(override)
        base = sum(int(x) for x in P) if isinstance(P, np.ndarray) else sum(P)
        self._total = F * base + sum(w - F * _num(P[v])
                                     for v, w in self.override.items())

    def total(self):
        return self._total

    def weight(self, v):
        if v in self.override:
            return self.override[v]
        return self.F * _num(self.P[v])

    def outcomes(self):
        out = []
        for v in range(len(self.P)):
            w = self.weight(v)
            if w > 0:
                out.append((v, w))
        return out

    def pick(self, t):
        """Smallest id whose inclusive prefix weight exceeds ``t``.  The prefix
        is non-decreasing, so a bisection over ids finds it; the prefix at an
        id is F * (sum of P up to it) corrected by the overridden tokens at or
        below it."""
        V = len(self.P)
        if isinstance(self.P, np.ndarray):
            cum = np.cumsum(self.P.astype(np.int64))      # exact: < 2^31 each, V < 2^18
        else:
            cum = np.cumsum(np.asarray(self.P, dtype=object))
        keys = sorted(self.override)
        corr = list(itertools.accumulate(self.override[u] - self.F * _num(self.P[u])
                                         for u in keys))

        def prefix(v):
            k = bisect.bisect_right(keys, v)
            return self.F * int(cum[v]) + (corr[k - 1] if k else 0)

        lo, hi = 0, V - 1
        assert prefix(hi) > t, "target beyond the total weight"
        while lo < hi:
            mid = (lo + hi) // 2
            if prefix(mid) > t:
                hi = mid
            else:
                lo = mid + 1
        return lo


# ---------------------------------------------------------------------------
# per-node draft distributions (Sec. 3.2, App. C.1, Sec. 5.4)
# ---------------------------------------------------------------------------

@dataclass
class NodeDist:
    """Draft-side quantities at one expanded node.

    support  token ids of the draft support, in rank order x_1, x_2, ...
             (construction probability descending, token id ascending)
    w1       construction weights (untempered q) in the same order
    s1       total construction weight, q(x_i) = w1[i] / s1: the sum of w1
             (or of every token's weight, for the whole-vocabulary reading)
    tail     q~ restricted to the support minus the top-m tokens, as an
             ExplicitDist of tempered weights; q~(v) = weight / total
    """
    support: list
    w1: list
    s1: object
    tail: ExplicitDist


def rank_order(ids, weights):
    """Ranks by (weight descending, token id ascending) -- the paper sorts
    by draft probability and leaves ties open; id order is this reading.
    Integer weights are ordered by a library sort on the same key."""
    if all(isinstance(x, (int, np.integer)) for x in weights):
        w = np.asarray(weights, dtype=np.int64)
        return np.lexsort((np.asarray(ids, dtype=np.int64), -w)).tolist()
    return sorted(range(len(ids)), key=lambda i: (-weights[i], int(ids[i])))


class UndefinedRow(ValueError):
    """A logit row on which the method is undefined."""


def _check_tail_reference(l_ref):
    """q~_T = q_T / z is evaluated relative to x_{m+1}'s logit; a masked
    token (logit -inf, probability 0 after the truncation of Sec. 3.2) there
    leaves it without a reference (and z may vanish): undefined."""
    if not np.float32(l_ref) > -np.inf:
        raise UndefinedRow("x_{m+1} has logit -inf")


def node_dist_from_logits(logits, m, T, support_size=0, construct_tempered=False,
                          model="canonical", construct_full=False):
    """Build the node's distributions from one row of draft logits.

    support_size S > 0 truncates the logits to the S largest entries (ties by
    lower id) before the softmax (Sec. 3.2); 0 keeps the full vocabulary.
    The construction distribution q is untempered unless
    ``construct_tempered`` (Sec. 5.4).  The tail q~ = q_T / z on the support
    minus x_1..x_m (App. C.1) is evaluated relative to the logit of x_{m+1},
    so its largest weight is 2**30 and its total never vanishes.  Y ~ q~ is
    drawn by inverse CDF over the tail in rank order (x_{m+1}, x_{m+2}, ...)
    when S > 0, and over token ids when the support is the vocabulary.

    ``construct_full``: the other reading of the sparse mode, where the
    truncation touches only the sampled token (Sec. 5.5, discussion of
    Table 5): the construction softmax runs over the whole vocabulary (its
    total s1 sums every token's weight; the support's weights and order are
    the same), while the tail q~ stays on the support."""
    l = np.asarray(logits, dtype=np.float32)
    V = l.shape[0]
    ids = np.arange(V, dtype=np.int64)
    # a sparse node samples Y over its tail in rank order, a dense one over
    # token ids (reading of the inverse CDF's order)
    ranked = bool(support_size and support_size > 0)
    order = np.lexsort((ids, -l.astype(np.float64)))
    if support_size and support_size < V:
        order = order[:support_size]
    sup = order
    ref = l[sup[0]]
    Tc = T if construct_tempered else 1.0
    if model == "canonical":
        wa = numerics.canonical_weights(l[sup], ref, Tc)
        r = np.lexsort((sup, -wa))                 # (weight desc, id asc)
        sup_r = sup[r]
        support = sup_r.tolist()
        w1 = wa[r].tolist()
        s1 = int(wa.sum())
        if construct_full and len(sup) < V:
            s1 = int(numerics.canonical_weights(l, ref, Tc).sum())
        tail_np = sup_r[m:]
        _check_tail_reference(l[tail_np[0]])
        q = numerics.canonical_weights(l[tail_np], l[tail_np[0]], T)
        return NodeDist(support, w1, s1, ExplicitDist(tail_np, q, ranked=ranked))
    else:
        w = numerics.fp64_weights(l[sup], ref, Tc)
        r = rank_order(list(sup), w)
        support = [int(sup[i]) for i in r]
        w1 = [w[i] for i in r]
    s1 = sum(w1)
    if construct_full and len(sup) < V:
        if model == "canonical":
            s1 = sum(int(x) for x in numerics.canonical_weights(l, ref, Tc))
        else:
            s1 = sum(numerics.fp64_weights(l, ref, Tc))
    tail_ids = support[m:]
    ref_t = l[tail_ids[0]]
    _check_tail_reference(ref_t)
    if model == "canonical":
        q = numerics.canonical_weights(l[tail_ids], ref_t, T).tolist()
    else:
        q = numerics.fp64_weights(l[tail_ids], ref_t, T)
    return NodeDist(support, w1, s1, ExplicitDist(tail_ids, q, ranked=ranked))


def node_dist_from_weights(ids, w1, q_tail=None, m=1):
    """A node given directly by construction weights (and optionally tempered
    tail weights; by default the tail of w1 itself, i.e. T = 1)."""
    r = rank_order(ids, w1)
    support = [int(ids[i]) for i in r]
    ws = [w1[i] for i in r]
    tail_ids = support[m:]
    if q_tail is None:
        q = ws[m:]
    else:
        q = [q_tail[int(v)] for v in tail_ids]
    return NodeDist(support, ws, sum(ws), ExplicitDist(tail_ids, q))


def target_weights(logits, T, model="canonical"):
    """p = softmax(target / T) over the whole vocabulary (verification never
    truncates p); weights relative to the row maximum."""
    l = np.asarray(logits, dtype=np.float32)
    ref = l.max()
    if not ref > -np.inf:
        raise UndefinedRow("target row has no finite logit")
    if model == "canonical":
        return numerics.canonical_weights(l, ref, T)
    return numerics.fp64_weights(l, ref, T)


# ---------------------------------------------------------------------------
# the hybrid candidate pool (Sec. 3.2; App. C.1)
# ---------------------------------------------------------------------------

def as_prob(num, den):
    """A probability reported in fp64: the correctly rounded quotient."""
    if isinstance(num, Fraction) or isinstance(den, Fraction):
        return float(Fraction(num) / Fraction(den))
    return int(num) / int(den)


def make_pool(nd, K, m, y, eps=2.0 ** -40, proxy_rule="rheo", adhoc_proxy=None):
    """The K slots of one parent's pool given the sampled token ``y``.

    Returns [(slot, token, kind, proxy, qtrue)], slots 1..K in the order
    top-m leads, Y, fills.  Leads and fills carry q(x) as proxy; Y carries
    min{q(x_m), z} with z = 1 - sum_{i<=m} q(x_i) (App. C.1), or q(x_1) + eps
    when m = 0 (Sec. 3.2), capped at 1 so that path scores never grow
    (Lemma 2).  ``qtrue`` is q~(Y) for the sampled slot and q(x) otherwise.
    ``proxy_rule='adhoc'`` replaces Y's proxy by the fixed ``adhoc_proxy``
    (the counterexample of Table 1; negative control only)."""
    x, w1, s1 = nd.support, nd.w1, nd.s1
    pool = []
    for i in range(m):
        p = as_prob(w1[i], s1)
        pool.append([i + 1, x[i], LEAD, p, p])
    if proxy_rule == "adhoc":
        py = float(adhoc_proxy)
    elif m >= 1:
        z_num = s1 - sum(w1[:m])
        py = as_prob(min(w1[m - 1], z_num), s1)
    else:
        py = min(1.0, as_prob(w1[0], s1) + eps)
    qt = as_prob(nd.tail.weight(y), nd.tail.total())
    pool.append([m + 1, y, SAMPLED, py, qt])
    fills = list(itertools.islice(((v, w) for v, w in zip(x[m:], w1[m:]) if v != y),
                                  K - m - 1))
    for j, (v, w) in enumerate(fills):
        p = as_prob(w, s1)
        pool.append([m + 2 + j, v, FILL, p, p])
    return pool


def make_topk_pool(nd, K):
    """Pure top-K pool of the EAGLE baseline (Sec. 2.1): no sampled slot."""
    out = []
    for i in range(min(K, len(nd.support))):
        p = as_prob(nd.w1[i], nd.s1)
        out.append([i + 1, nd.support[i], LEAD, p, p])
    return out


# ---------------------------------------------------------------------------
# the draft tree: expand-then-rerank, then global pruning
# ---------------------------------------------------------------------------

@dataclass
class Node:
    uid: int
    parent: int          # uid of the parent, -1 for the root
    depth: int
    slot: int            # 1..K, 0 for the root
    token: int           # -1 for the root
    kind: int
    proxy: float
    qtrue: float
    score: float         # product of proxies root -> node (App. C.1)
    path: tuple          # slot indices root -> node ("left-to-right" order)
    dist: NodeDist = None    # set when the node is expanded
    expanded: bool = False
    children: list = field(default_factory=list)


def priority(node):
    """Global ranking key (App. C.1): path score descending, then depth
    ascending, then left-to-right sibling order (the slot path)."""
    return (-node.score, node.depth, node.path)


@dataclass
class TreeConfig:
    K: int
    m: int
    depth: int
    n_expand: int = None
    support: int = 0
    construct_tempered: bool = False
    construct_full: bool = False  # construction over the whole vocabulary, sparse tail
    eps: float = 2.0 ** -40
    mode: str = "rheo"           # "rheo" or "topk" (pure top-K baseline)
    verifier: str = "rheo"       # "rheo" (Algorithm 1) or "rrsw" (App. D.2 baseline)
    proxy_rule: str = "rheo"     # "adhoc" only for the negative control
    adhoc_proxy: float = None
    model: str = "canonical"

    def __post_init__(self):
        if self.n_expand is None:
            self.n_expand = self.K


def build_tree(cfg, T, draft_dist, seq=0):
    """Expand-then-rerank (Sec. 2.1) with Rheo pools; a generator that
    yields one Cat request per expanded node and returns the list of nodes
    indexed by uid.  ``draft_dist(node, nodes)`` returns the NodeDist of the
    draft model at ``node`` (the synthetic stand-in for a draft forward).

    uids: the root is 0; each level's children are numbered in frontier order
    (frontier = the selected parents ranked by priority), slots in order."""
    root = Node(0, -1, 0, 0, -1, LEAD, 1.0, 1.0, 1.0, ())
    nodes = [root]
    frontier = [root]
    for d in range(cfg.depth):
        level = []
        for parent in frontier:
            nd = draft_dist(parent, nodes)
            parent.dist = nd
            parent.expanded = True
            if cfg.mode == "topk":
                pool = make_topk_pool(nd, cfg.K)
            else:
                y = yield Cat(DRAFT, parent.uid, nd.tail)
                pool = make_pool(nd, cfg.K, cfg.m, y, cfg.eps, cfg.proxy_rule,
                                 cfg.adhoc_proxy)
            for slot, tok, kind, proxy, qtrue in pool:
                child = Node(len(nodes), parent.uid, d + 1, slot, tok, kind,
                             proxy, qtrue, parent.score * proxy,
                             parent.path + (slot,))
                nodes.append(child)
                parent.children.append(child.uid)
                level.append(child)
        if d + 1 < cfg.depth:
            frontier = sorted(level, key=priority)[:cfg.n_expand]
    return nodes


def frontier_of_level(nodes, depth, n_expand):
    """The nodes selected for expansion at ``depth`` (ranked)."""
    cands = [n for n in nodes if n.depth == depth]
    return sorted(cands, key=priority)[:n_expand]


@dataclass
class PrunedTree:
    order: list          # pruned index -> uid (index 0 is the root)
    parent: list         # pruned index -> pruned index of the parent
    children: list       # pruned index -> [pruned indices], slot order
    sampled: list        # pruned index -> position of the sampled child or -1


def tree_mask(nodes, pt):
    """What the target model needs to score the pruned tree in one forward
    pass (Sec. 1; Sec. 2.1: the drafted paths are verified in parallel):
    mask[i][j] = 1 iff pruned node j lies on the path from the root to
    pruned node i (i itself included), and the depth of every pruned node
    (the root 0), i.e. its position after the prefix."""
    n = len(pt.order)
    mask = [[0] * n for _ in range(n)]
    depth = [0] * n
    for i in range(n):
        j, d = i, 0
        while j != -1:
            mask[i][j] = 1
            j = pt.parent[j]
            d += 1
        depth[i] = d - 1
        assert depth[i] == nodes[pt.order[i]].depth
    return mask, depth


def prune(nodes, R):
    """Keep the R best non-root nodes under ``priority`` (App. C.1).  The
    root is not counted in R (App. C.3, base case: T_1 is one depth-1
    node).  Pruned indices follow the rank order."""
    ranked = sorted(nodes[1:], key=priority)[:R]
    order = [0] + [n.uid for n in ranked]
    index = {uid: i for i, uid in enumerate(order)}
    parent = [-1]
    for n in ranked:
        assert n.parent in index, "pruned tree is not ancestor-closed"
        parent.append(index[n.parent])
    children = [[] for _ in order]
    for i in range(1, len(order)):
        children[parent[i]].append(i)
    sampled = []
    for i, ch in enumerate(children):
        ch.sort(key=lambda j: nodes[order[j]].slot)
        s = -1
        for pos, j in enumerate(ch):
            if nodes[order[j]].kind == SAMPLED:
                s = pos
        sampled.append(s)
    return PrunedTree(order, parent, children, sampled)


# ---------------------------------------------------------------------------
# RheoVerification (Algorithm 1), layer by layer (Thm. 1)
# ---------------------------------------------------------------------------

def _candidate_tests(nodes, pt, cand, level, r, z_rem):
    """Sequential tests of ``cand`` (pruned indices, slot order) under the
    residual ``r`` of mass ``z_rem``: accept the first candidate u with
    eta <= r(u); a rejected candidate gets r(u) = 0 (renormalised).  Yields
    Bern requests; returns (accepted index or None, remaining mass)."""
    for j in cand:
        tok = nodes[pt.order[j]].token
        nv = r.weight(tok)
        ok = yield Bern(VERIFY, 32 * level + nodes[pt.order[j]].slot, nv, z_rem)
        if ok:
            return j, z_rem
        r.override[tok] = 0
        r._total -= nv
        z_rem -= nv
    return None, z_rem


def verify(nodes, pt, target_P, verifier="rheo"):
    """Walk the pruned tree from the root.  ``target_P(i)`` returns the
    target weights P over the vocabulary at pruned node i (p = P / sum P).
    Yields Bern / Cat requests; returns (accepted tokens, final token).

    Per layer (Algorithm 1): candidates C = children in slot order, s the
    sampled child's position.  If s != -1: accept u_s iff
    eta <= p(u_s) / q~(u_s); otherwise drop u_s and set
    r = norm(max(0, p - q~)).  If s == -1: r = p.  Then for each remaining
    candidate in order: accept iff eta <= r(u_i), else r(u_i) = 0 and
    renormalise.  If none is accepted, emit u* ~ r.  With integer weights
    r(v) = N_v / Z and the tests are exact integer comparisons.

    ``verifier='rrsw'``: the recursive rejection baseline of App. D.2, which
    keeps the pool but tests the sampled child after the leads: the leads
    (the candidates before u_s) under p, then u_s under the remaining
    target r (accept iff eta <= r(u_s) / q~(u_s)), then, after a rejection,
    the fills under norm(max(0, r - q~)).  Without a sampled child both
    verifiers are the same sequential test under p."""
    accepted = []
    cur = 0
    level = 0
    while True:
        P = target_P(cur)
        Sp = int(P.sum()) if isinstance(P, np.ndarray) else sum(P)
        cand = list(pt.children[cur])
        if not cand:
            u = yield Cat(FINAL, level, ResidualDist(P, 1, {}))
            return accepted, u
        node_cur = nodes[pt.order[cur]]
        s = pt.sampled[cur]
        F = 1
        override = {}
        z_y = Sp                   # mass of the target r when u_s is tested
        if s != -1 and verifier == "rrsw":
            r = ResidualDist(P, 1, {})
            hit, z_y = yield from _candidate_tests(nodes, pt, cand[:s], level, r, Sp)
            if hit is not None:
                accepted.append(nodes[pt.order[hit]].token)
                cur = hit
                level += 1
                continue
            override = dict(r.override)          # the rejected leads, zeroed
            cand = cand[s:]
            s = 0
        if s != -1:
            tail = node_cur.dist.tail
            Zq = tail.total()
            y_idx = cand[s]
            Y = nodes[pt.order[y_idx]].token
            ok = yield Bern(VERIFY, 32 * level, _num(P[Y]) * Zq,
                            tail.weight(Y) * z_y)
            if ok:
                accepted.append(Y)
                cur = y_idx
                level += 1
                continue
            del cand[s]
            # r = norm(max(0, r - q~)): numerators P_v Zq - Q_v z_y over
            # z_y Zq (rejected leads stay at 0)
            F = Zq
            for v, qv in zip(tail.ids, tail.weights):
                override[v] = max(0, _num(P[v]) * Zq - qv * z_y)
        r = ResidualDist(P, F, override)
        hit, _ = yield from _candidate_tests(nodes, pt, cand, level, r, r.total())
        if hit is not None:
            accepted.append(nodes[pt.order[hit]].token)
            cur = hit
            level += 1
            continue
        u = yield Cat(FINAL, level, r)
        return accepted, u


def rheo_step(cfg, T, R, draft_dist, target_P, seq=0):
    """One full step for one sequence: build, prune, verify.  Returns
    (nodes, pruned tree, accepted tokens, final token)."""
    nodes = yield from build_tree(cfg, T, draft_dist, seq)
    pt = prune(nodes, R)
    acc, u = yield from verify(nodes, pt, target_P, cfg.verifier)
    return nodes, pt, acc, u
