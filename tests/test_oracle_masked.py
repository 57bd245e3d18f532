"""Masked vocabulary (logits of -inf) in the oracle.

Sec. 3.2 truncates the draft distribution by setting logits to -inf, and
engines mask tokens the same way (padded vocabularies, constrained
decoding).  A masked token has probability 0.  Pins:
  * the limit: a masked token behaves exactly like a logit so far below the
    rest that its weight underflows to 0 (every distribution the node and
    the target define is the same, token for token);
  * Thm. 1 by exact enumeration with masks shared by draft and target,
    masks of the draft alone (q = 0 where p > 0) and of the target alone
    (the draft proposes tokens p forbids): the output is p, masked tokens
    are never emitted, and every sequence p allows is reachable;
  * the undefined cases raise: a draft row whose x_{m+1} is masked (q~_T has
    no reference) and a target row with no finite logit.
"""

import itertools
import zlib
from fractions import Fraction

import numpy as np
import pytest
import torch

import synth
from oracle import numerics, rheo
from test_oracle_pins import _logits_fn, _multi_step_dist, _target_seq_prob

F = Fraction
NEG = np.float32(-1e30)


def _mask(rng, V, frac, keep):
    """A random mask with at least ``keep`` tokens left (lowest masked ids
    unmasked first)."""
    mk = rng.random(V) < frac
    for v in range(V):
        if (~mk).sum() >= keep:
            break
        mk[v] = False
    return mk


def _nd_equal(a, b):
    assert a.support == b.support
    assert a.w1 == b.w1 and a.s1 == b.s1
    assert list(a.tail.ids) == list(b.tail.ids)
    assert [int(x) for x in a.tail.weights] == [int(x) for x in b.tail.weights]


@pytest.mark.parametrize("seed", range(24))
def test_masked_equals_underflow_limit(seed):
    rng = np.random.default_rng(7000 + seed)
    V = int(rng.integers(6, 40))
    m = int(rng.integers(0, 3))
    S = [0, 4, 8, 16][seed % 4]
    T = [0.5, 1.0, 1.7][seed % 3]
    frac = [0.2, 0.6, 0.9][seed % 3]
    l = (rng.normal(0, 2.0, V)).astype(np.float32)
    # enough finite tokens that x_{m+1} is finite in both rows
    mk = _mask(rng, V, frac, m + 1)
    lm, ln = l.copy(), l.copy()
    lm[mk] = -np.inf
    ln[mk] = NEG
    for tempered, full in ((False, False), (True, False), (False, True)):
        a = rheo.node_dist_from_logits(lm, m, T, S, tempered, "canonical", full)
        b = rheo.node_dist_from_logits(ln, m, T, S, tempered, "canonical", full)
        _nd_equal(a, b)
        # masked tokens carry weight 0 wherever they appear
        for v, w in zip(a.support, a.w1):
            if mk[v]:
                assert w == 0
        for v, w in zip(a.tail.ids, a.tail.weights):
            if mk[v]:
                assert w == 0
    pa = rheo.target_weights(lm, T)
    pb = rheo.target_weights(ln, T)
    assert np.array_equal(pa, pb) and not pa[mk].any()


def test_masked_support_fills_with_zero_weight_ids():
    # fewer finite logits than the support: the support ends with masked
    # tokens, weight 0, in id order (the rank by (weight desc, id asc))
    V, S, m = 12, 6, 1
    l = np.full(V, -np.inf, np.float32)
    l[[9, 3, 7]] = [1.0, 0.5, 0.25]
    nd = rheo.node_dist_from_logits(l, m, 1.0, S)
    assert nd.support == [9, 3, 7, 0, 1, 2]
    assert nd.w1[3:] == [0, 0, 0] and all(w > 0 for w in nd.w1[:3])
    assert sorted(nd.tail.ids) == [0, 1, 2, 3, 7]
    assert nd.tail.weight(3) == 2 ** numerics.WSHIFT     # x_2, the reference
    assert 0 < nd.tail.weight(7) < nd.tail.weight(3)
    assert [nd.tail.weight(v) for v in (0, 1, 2)] == [0, 0, 0]


def _masked_logits_fn(seed, V, mode, m):
    """_logits_fn with masks: 'shared' (the same mask on the draft and the
    target row of a prefix), 'draft' (draft only) or 'target' (target only);
    the draft keeps >= m + 1 tokens, the target >= 1."""
    base = _logits_fn(seed, V)
    cache = {}

    def f(role, prefix):
        k = (role, prefix)
        if k not in cache:
            rng = np.random.default_rng([seed, 99, len(prefix)] + [int(x) for x in prefix])
            shared = _mask(rng, V, 0.4, m + 1)
            own = _mask(rng, V, 0.4, m + 1)
            if mode == "shared":
                mk = shared
            elif mode == "draft":
                mk = own if role == "d" else np.zeros(V, bool)
            else:
                mk = own if role == "t" else np.zeros(V, bool)
            row = base(role, prefix).copy()
            row[mk] = -np.inf
            cache[k] = row
        return cache[k]
    return f


MASKED_CASES = [
    # V, K, m, depth, R, T, support, mode, verifier, model
    (5, 3, 1, 2, 4, 1.0, 0, "shared", "rheo", "canonical"),
    (5, 3, 1, 2, 4, 1.0, 0, "draft", "rheo", "canonical"),
    (5, 3, 1, 2, 4, 1.0, 0, "target", "rheo", "canonical"),
    (6, 3, 1, 2, 5, 0.7, 4, "shared", "rheo", "canonical"),
    (6, 4, 2, 2, 6, 1.0, 5, "draft", "rheo", "canonical"),
    (5, 3, 0, 2, 4, 1.3, 0, "target", "rheo", "canonical"),
    (5, 3, 1, 2, 4, 1.0, 3, "shared", "rrsw", "canonical"),
    (5, 3, 1, 2, 4, 1.0, 0, "target", "rrsw", "canonical"),
    (5, 3, 1, 2, 4, 1.0, 0, "shared", "rheo", "fp64"),
]


@pytest.mark.parametrize("case", MASKED_CASES)
def test_thm1_lossless_with_masks(case):
    V, K, m, D, R, T, S, mode, verifier, model = case
    L = 2
    seed = zlib.crc32(repr(case).encode()) & 0xFFFF
    lf = _masked_logits_fn(seed, V, mode, m)
    cfg = rheo.TreeConfig(K=K, m=m, depth=D, n_expand=min(K, 2), support=S, model=model,
                          verifier=verifier)
    dist = _multi_step_dist(cfg, T, R, L, lf, model)
    assert sum(dist.values()) == 1
    for seq, prob in dist.items():
        assert prob == _target_seq_prob(seq, T, lf, model), seq
        assert prob > 0
    # exactly the sequences p allows are emitted (masked tokens never are)
    allowed = [s for s in itertools.product(range(V), repeat=L)
               if _target_seq_prob(s, T, lf, model) > 0]
    assert sorted(dist) == sorted(allowed)
    assert len(allowed) < V ** L or mode == "draft"


def test_undefined_rows_raise():
    V = 10
    l = np.full(V, -np.inf, np.float32)
    l[4] = 0.0
    # m = 1: x_2 is masked, so q~_T has no reference token
    with pytest.raises(rheo.UndefinedRow):
        rheo.node_dist_from_logits(l, 1, 1.0, 0)
    with pytest.raises(rheo.UndefinedRow):
        rheo.node_dist_from_logits(l, 1, 1.0, 4, model="fp64")
    # m = 0: x_1 is the reference; defined, and the tail is the one token
    nd = rheo.node_dist_from_logits(l, 0, 1.0, 4)
    assert nd.support == [4, 0, 1, 2] and nd.tail.total() == 2 ** numerics.WSHIFT
    with pytest.raises(rheo.UndefinedRow):
        rheo.target_weights(np.full(V, -np.inf, np.float32), 1.0)


def test_synth_masks():
    w = synth.WORKLOADS["llama2"].with_(mask=0.75, mask_tail=300, mask_target=0.1)
    keys = [synth.root_key(w, b, 0) for b in range(4)]
    d = synth.as_fp32_numpy(synth.draft_rows(w, keys))
    t = synth.as_fp32_numpy(synth.target_rows(w, keys, [0.7] * 4))
    fin_d, fin_t = np.isfinite(d), np.isfinite(t)
    assert not fin_d[:, -300:].any()
    assert abs(fin_d[:, :-300].mean() - 0.25) < 0.01
    assert not (fin_t & ~fin_d).any()               # a draft mask holds in the target
    assert abs((fin_d & ~fin_t).sum() / fin_d.sum() - 0.1) < 0.02
    assert (d[fin_d] > -np.inf).all() and not np.isnan(d).any() and not np.isnan(t).any()
    # bf16 rounding keeps -inf
    w3 = synth.WORKLOADS["llama3"].with_(mask=0.5)
    r = synth.draft_rows(w3, keys[:1])
    neg = r.view(torch.int16) == -128                # bf16 0xFF80
    assert torch.equal(neg, r.float() == -np.inf)
    assert abs(neg.float().mean().item() - 0.5) < 0.01
