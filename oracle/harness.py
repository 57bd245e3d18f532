"""Runs the oracle on the synthetic workloads.  TEST INFRASTRUCTURE ONLY.

A node's draft row and target row are generated from its path key (the
prefix key extended by the node's tokens) by the shared input module
``synth``; everything else is the oracle's own arithmetic.
"""

import numpy as np

import synth
from . import rheo
from .drivers import run_philox


def tree_config(w, **over):
    kw = dict(K=w.K, m=w.m, depth=w.depth, n_expand=w.n_expand,
              support=w.support, construct_tempered=w.construct_tempered,
              construct_full=w.construct_full,
              eps=w.eps_m0, mode="topk" if w.method == "topk" else "rheo",
              verifier="rrsw" if w.method == "rrsw" else "rheo")
    kw.update(over)
    return rheo.TreeConfig(**kw)


def node_key(nodes, uid, root):
    path = []
    while uid > 0:
        path.append(nodes[uid].token)
        uid = nodes[uid].parent
    key = root
    for tok in reversed(path):
        key = synth.child_key(key, tok)
    return key


def oracle_step(w, b, step, T=None, trace=None, model="canonical", cfg=None,
                row_cache=None):
    """One step of sequence ``b`` of workload ``w`` under the oracle.
    Returns (nodes, pruned tree, accepted tokens, final token).
    ``row_cache`` (a dict) memoises generated rows by node key, so that a
    second run times the method without the synthetic-input generation."""
    T = w.T if T is None else T
    cfg = cfg or tree_config(w, model=model)
    root = synth.root_key(w, b, step)
    sig = synth.seq_sigma_t(w, b)

    cache = {} if row_cache is None else row_cache

    def draft_dist(node, nodes):
        key = node_key(nodes, node.uid, root)
        if ("d", key) not in cache:
            cache[("d", key)] = synth.as_fp32_numpy(synth.draft_rows(w, [key]))[0]
        row = cache[("d", key)]
        return rheo.node_dist_from_logits(row, cfg.m, T, cfg.support,
                                          cfg.construct_tempered, model,
                                          cfg.construct_full)

    holder = {}

    def target_P(i):
        nodes, pt = holder["nodes"], holder["pt"]
        key = node_key(nodes, pt.order[i], root)
        if ("t", key) not in cache:
            cache[("t", key)] = synth.as_fp32_numpy(synth.target_rows(w, [key], [sig]))[0]
        row = cache[("t", key)]
        return rheo.target_weights(row, T, model)

    def process():
        nodes = yield from rheo.build_tree(cfg, T, draft_dist, b)
        pt = rheo.prune(nodes, w.R)
        holder["nodes"], holder["pt"] = nodes, pt
        acc, u = yield from rheo.verify(nodes, pt, target_P, cfg.verifier)
        return nodes, pt, acc, u

    return run_philox(process(), synth.step_rng_key(w, step), b, trace)


def node_table(nodes):
    """The unpruned tree as arrays in uid order (root included)."""
    return {
        "token": np.array([n.token for n in nodes], dtype=np.int64),
        "parent": np.array([n.parent for n in nodes], dtype=np.int64),
        "depth": np.array([n.depth for n in nodes], dtype=np.int64),
        "slot": np.array([n.slot for n in nodes], dtype=np.int64),
        "kind": np.array([n.kind for n in nodes], dtype=np.int64),
        "proxy": np.array([n.proxy for n in nodes], dtype=np.float64),
        "qtrue": np.array([n.qtrue for n in nodes], dtype=np.float64),
        "score": np.array([n.score for n in nodes], dtype=np.float64),
    }
