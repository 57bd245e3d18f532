"""Pins of the oracle's temperature handling and of its node records against
an independent fp64 computation (numpy ``exp`` and ``argmax``), written here
without calling the oracle's weight functions.

* Verification's p is softmax(target / T) over the whole vocabulary
  (Algorithm 1; Sec. 5.4 applies T to sampling and verification): the
  oracle's quantised p must match the fp64 softmax of l / T within the
  quantisation bound, and must not match it at another temperature.
* At T -> 0 every softmax is one-hot (Sec. 5.4): RheoVerification then
  accepts a drafted child iff it is the target's argmax at its parent, and
  the emitted token after the accepted path is the target's argmax there.
* Every node record (proxy, true probability, path score; App. C.1, Sec.
  3.2) agrees with the same quantities computed in fp64 from the node's own
  draft row, within max(1e-5 q, 2^-28).
"""

import numpy as np
import pytest

import synth
from oracle import rheo
from oracle.harness import oracle_step

W = synth.WORKLOADS


def _softmax64(l, T):
    x = np.asarray(l, dtype=np.float64)
    x = (x - x.max()) / float(np.float32(T))
    e = np.exp(x)
    return e / e.sum()


def _rows(w, n, seed):
    keys = [synth.splitmix64(seed * 7919 + i) for i in range(n)]
    return synth.as_fp32_numpy(synth.target_rows(w, keys, [synth.seq_sigma_t(w, 0)] * n))


# --------------------------------------------------------------------------
# p = softmax(target / T) in verification
# --------------------------------------------------------------------------

@pytest.mark.parametrize("T", [0.5, 0.8, 2.0])
@pytest.mark.parametrize("wl", ["llama2", "large"])
def test_target_weights_are_softmax_at_T(T, wl):
    w = W[wl].with_(V=20000)
    for row in _rows(w, 4, 11):
        P = rheo.target_weights(row, T).astype(np.float64)
        p_hat = P / P.sum()
        p = _softmax64(row, T)
        # per weight: < 5e-6 relative plus one unit of 2^-30 (relative to the
        # maximum); the total adds V units
        bound = 1e-5 * p + (2.0 + len(row)) * 2.0 ** -30 / (P.sum() / 2.0 ** 30)
        assert np.all(np.abs(p_hat - p) <= bound), float(np.max(np.abs(p_hat - p) / bound))


@pytest.mark.parametrize("T", [0.5, 2.0])
def test_target_temperature_pin_has_power(T):
    """The same comparison fails when p is taken at T = 1 instead of T."""
    w = W["llama2"].with_(V=5000)
    row = _rows(w, 1, 3)[0]
    P = rheo.target_weights(row, 1.0).astype(np.float64)
    p = _softmax64(row, T)
    assert np.max(np.abs(P / P.sum() - p)) > 1e-3


# --------------------------------------------------------------------------
# T -> 0: verification is a greedy match against the target argmax
# --------------------------------------------------------------------------

def _node_key(nodes, uid, root):
    toks = []
    while uid > 0:
        toks.append(nodes[uid].token)
        uid = nodes[uid].parent
    k = root
    for t in reversed(toks):
        k = synth.child_key(k, t)
    return k


@pytest.mark.parametrize("m", [0, 1, 2])
@pytest.mark.parametrize("wl", ["tiny", "small_zipf"])
def test_greedy_verification_at_low_temperature(m, wl):
    T = 1e-4
    if wl == "tiny":
        w = W["tiny"].with_(K=4, m=m, R=10)
    else:
        w = W["llama2"].with_(name="small_zipf", V=3000, K=4, m=m, depth=3, R=12)
    # logits closer than this may leave more than one token with weight > 0
    gap_min = 32.0 * T
    checked = 0
    for step in range(12):
        nodes, pt, acc, u = oracle_step(w, 0, step, T=T)
        root = synth.root_key(w, 0, step)
        sig = synth.seq_sigma_t(w, 0)

        def target_row(i):
            key = _node_key(nodes, pt.order[i], root)
            return synth.as_fp32_numpy(synth.target_rows(w, [key], [sig]))[0]

        cur, want, ok = 0, [], True
        while True:
            row = target_row(cur).astype(np.float64)
            top2 = np.sort(row)[-2:]
            if top2[1] - top2[0] < gap_min:
                ok = False
                break
            a = int(np.argmax(row))
            kids = {nodes[pt.order[j]].token: j for j in pt.children[cur]}
            if a in kids:
                want.append(a)
                cur = kids[a]
            else:
                break
        if not ok:
            continue
        checked += 1
        assert list(acc) == want and u == a, (step, acc, want, u, a)
        # the sampled token of every expanded node is x_{m+1}
        for n in nodes:
            if n.expanded:
                y = [nodes[c] for c in n.children if nodes[c].kind == rheo.SAMPLED][0]
                row = synth.as_fp32_numpy(synth.draft_rows(w, [_node_key(nodes, n.uid, root)]))[0]
                order = np.lexsort((np.arange(len(row)), -row.astype(np.float64)))
                assert y.token == int(order[m])
    assert checked >= 8


# --------------------------------------------------------------------------
# node records against fp64
# --------------------------------------------------------------------------

def _fp64_pool(row, w, T, y):
    """Leads, Y and fills of a node with their proxies and true
    probabilities, from its draft row in fp64 (Sec. 3.2; App. C.1)."""
    l = np.asarray(row, dtype=np.float64)
    V = len(l)
    order = np.lexsort((np.arange(V), -l))
    S = w.support if (w.support and w.support < V) else V
    sup = order[:S]
    Tc = T if w.construct_tempered else 1.0
    e1 = np.exp((l[sup] - l[sup[0]]) / Tc)
    q1 = e1 / e1.sum()
    m, K = w.m, w.K
    out = []
    for i in range(m):
        out.append((int(sup[i]), q1[i], q1[i]))
    if m >= 1:
        py = min(q1[m - 1], 1.0 - q1[:m].sum())
    else:
        py = min(1.0, q1[0] + w.eps_m0)
    tail = sup[m:]
    eT = np.exp((l[tail] - l[tail[0]]) / float(np.float32(T)))
    qt = eT / eT.sum()
    yi = int(np.nonzero(tail == y)[0][0])
    out.append((y, py, qt[yi]))
    rest = [(int(v), q1[m + i]) for i, v in enumerate(tail) if int(v) != y][:K - m - 1]
    out.extend((v, q, q) for v, q in rest)
    return out


def _close(a, b):
    return abs(a - b) <= max(1e-5 * abs(b), 2.0 ** -28)


@pytest.mark.parametrize("over", [
    dict(),
    dict(m=0),
    dict(m=2, K=5),
    dict(T=0.6),
    dict(T=0.6, construct_tempered=True),
    dict(T=1.5, support=0),
])
def test_node_records_match_fp64(over):
    kw = dict(name="rec", V=4000, K=4, depth=3, R=12)
    kw.update(over)
    w = W["llama2"].with_(**kw)
    T = w.T
    nrec = 0
    for step in range(3):
        nodes, pt, acc, u = oracle_step(w, 0, step)
        root = synth.root_key(w, 0, step)
        for n in nodes:
            if not n.expanded:
                continue
            row = synth.as_fp32_numpy(synth.draft_rows(w, [_node_key(nodes, n.uid, root)]))[0]
            kids = [nodes[c] for c in n.children]
            y = [c for c in kids if c.kind == rheo.SAMPLED][0].token
            want = _fp64_pool(row, w, T, y)
            assert [c.token for c in kids] == [t for t, _, _ in want]
            for c, (_, px, qt) in zip(kids, want):
                assert _close(c.proxy, px), (c.uid, c.proxy, px)
                assert _close(c.qtrue, qt), (c.uid, c.qtrue, qt)
                assert _close(c.score, n.score * px), (c.uid, c.score, n.score * px)
                nrec += 1
    assert nrec >= 3 * (w.K + (w.depth - 1) * w.K * w.K)
