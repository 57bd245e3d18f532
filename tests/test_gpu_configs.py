"""GPU parity at the workload sizes: every sequence of the batched shapes in
both modes, the long tiny run, the tempered construction reading, the
rheostat x temperature grid (Sec. 5.3, Sec. 5.4) and the T -> 0
degeneracy on the HIP path.

The oracle's results come from worker processes (``oracle_pool``) that run
while the GPU works; the comparison is the one of ``test_gpu_parity``:
topology, tokens, kinds, pruned tree, mask, accepted and final tokens
bit-exact, probabilities within 1e-5 relative (in fact bit-exact).
"""

import os

import numpy as np
import pytest
import torch

import synth
from oracle_pool import OraclePool

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS
INT_FIELDS = ("token", "parent", "depth", "slot", "kind")
FP_FIELDS = ("proxy", "qtrue", "score")


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2609_21827_amd import binding
    binding.load_library()
    return "cuda"


def gpu_steps(w, steps, T, dev, tree_kw=None, light=False):
    """Runs ``steps`` on one handle; per step the node records, pruned view,
    mask, depth and outputs as numpy arrays."""
    from paper_2609_21827_amd.driver import make_tree, run_step
    tree = make_tree(w, device=dev, **(tree_kw or {}))
    out = {}
    try:
        for i, step in enumerate(steps):
            if not light or i % 500 == 0:
                print(f"gpu {w.name} step={step} T={T}", flush=True)
            acc, alen, fin = run_step(tree, w, step, T=T, device=dev)
            rec = dict(nodes={k: v.cpu().numpy() for k, v in tree.read_nodes().items()})
            rec["ppar"], rec["ptok"] = (x.cpu().numpy() for x in tree.pruned_view())
            rec["mask"], rec["depth"] = (x.cpu().numpy() for x in tree.tree_mask())
            rec["acc"], rec["alen"], rec["fin"] = acc.numpy(), alen.numpy(), fin.numpy()
            out[step] = rec
        torch.cuda.synchronize()
        assert tree.device_error() == 0
    finally:
        tree.close()
    return out


def compare(w, gpu, orc, seqs, steps):
    for step in steps:
        g = gpu[step]
        for b in seqs:
            o = orc[(b, step)]
            ctx = (w.name, b, step)
            for k in INT_FIELDS:
                got = g["nodes"][k][b]
                assert np.array_equal(got, o["tab"][k]), (ctx, k, np.nonzero(got != o["tab"][k])[0][:8])
            for k in FP_FIELDS:
                got, want = g["nodes"][k][b], o["tab"][k]
                rel = np.abs(got - want) / np.maximum(np.abs(want), 1e-300)
                assert np.all(rel <= 1e-5), (ctx, k, float(rel.max()))
                assert np.array_equal(got, want), (ctx, k)
            assert list(g["ptok"][b]) == o["ptok"], ctx
            assert list(g["ppar"][b]) == o["ppar"], ctx
            assert np.array_equal(g["mask"][b], o["mask"]), ctx
            assert list(g["depth"][b]) == o["depth"], ctx
            n = int(g["alen"][b])
            assert list(g["acc"][b][:n]) == o["acc"], ctx
            assert all(x == -1 for x in g["acc"][b][n:]), ctx
            assert int(g["fin"][b]) == o["u"], ctx


def run_all(w, steps, dev, T=None, seqs=None, tree_kw=None, per_task=1, light=False):
    T = w.T if T is None else T
    seqs = list(range(w.B)) if seqs is None else seqs
    pool = OraclePool([(w, b, s, T) for s in steps for b in seqs], per_task=per_task)
    gpu = gpu_steps(w, steps, T, dev, tree_kw, light=light)
    orc = pool.results()
    print(f"  oracle done: {len(orc)} sequence-steps", flush=True)
    compare(w, gpu, orc, seqs, steps)
    return gpu, orc


# ---- the batched shapes, every sequence, both modes ----------------------

def test_batched_all_sequences(dev):
    run_all(W["batched"], [0, 1], dev)


def test_large_all_sequences(dev):
    w = W["large"]
    _, orc = run_all(w, [0, 1], dev)
    # the near one-hot peaks (5 % of nodes) were expanded on this path
    peaks = sum(synth.peaked(w, k) for o in orc.values() for k in o["expanded_keys"])
    assert peaks > 0


def test_batched_dense_all_sequences(dev):
    run_all(W["batched"].with_(name="batched_dense", support=0), [0], dev)


def test_large_dense_all_sequences(dev):
    w = W["large"].with_(name="large_dense", support=0)
    _, orc = run_all(w, [0], dev)
    assert sum(synth.peaked(w, k) for o in orc.values() for k in o["expanded_keys"]) > 0


# ---- cfg1 at its step count; cfg3 under the tempered construction --------

def test_tiny_long_run(dev):
    w = W["tiny"]
    run_all(w, list(range(w.steps)), dev, per_task=250, light=True)


@pytest.mark.parametrize("T", [0.6, 1.0])
def test_llama3_tempered_construction(dev, T):
    # the other reading of Sec. 5.4: the tree built on the tempered q
    run_all(W["llama3"].with_(name="llama3_tempered", construct_tempered=True), [0, 1], dev, T=T)


# ---- rheostat x temperature (Sec. 5.3, Sec. 5.4) --------------------------

@pytest.mark.parametrize("T", [0.2, 0.6, 1.0, 1.5])
@pytest.mark.parametrize("m", [0, 1, 2, 3])
def test_rheostat_grid(dev, m, T):
    w = W["headline"].with_(name=f"grid_m{m}", m=m, B=8, depth=4, R=30)
    run_all(w, [0], dev, T=T)


@pytest.mark.parametrize("m", [0, 3])
def test_rheostat_grid_dense(dev, m):
    w = W["llama2"].with_(name=f"grid_dense_m{m}", m=m, support=0, B=4, depth=4, R=30)
    run_all(w, [0], dev, T=0.2)


# ---- T -> 0 (Sec. 5.4, "Degeneracy asymmetry") ---------------------------

def _expanded_rows(w, nodes_b, root):
    """(uid, draft row) of every expanded node of one sequence's GPU tree."""
    tok, par = nodes_b["token"], nodes_b["parent"]
    keys = {0: root}
    for u in range(1, len(tok)):
        keys[u] = synth.child_key(keys[int(par[u])], int(tok[u]))
    exp = sorted({int(p) for p in par[1:] if p >= 0})
    rows = synth.as_fp32_numpy(synth.draft_rows(w, [keys[u] for u in exp]))
    return list(zip(exp, rows))


def test_low_temperature_degeneracy(dev):
    """At T = 1e-4 the sampled token is x_{m+1}; with m = 0 (and a tiny
    epsilon) the tree is the pure top-K tree bit for bit, with m = 1 it is
    not (the proxy min{q(x_1), z} replaces q(x_2))."""
    T = 1e-4
    base = W["llama2"].with_(name="t0", B=4, K=4, n_expand=4, depth=4, R=30,
                             eps_m0=2.0 ** -80)
    trees = {}
    for name, over in (("topk", dict(method="topk", m=1)), ("m0", dict(m=0)), ("m1", dict(m=1))):
        w = base.with_(name="t0_" + name, **over)
        gpu, _ = run_all(w, [0, 1, 2], dev, T=T)
        trees[name] = (w, gpu)
    differs = False
    for step in (0, 1, 2):
        ref = trees["topk"][1][step]["nodes"]
        for name in ("m0", "m1"):
            w, gpu = trees[name]
            nd = gpu[step]["nodes"]
            same = all(np.array_equal(nd[k], ref[k]) for k in ("token", "parent", "slot"))
            if name == "m0":
                assert same, step
            else:
                differs |= not same
            for b in range(w.B):
                nb = {k: v[b] for k, v in nd.items()}
                for uid, row in _expanded_rows(w, nb, synth.root_key(w, b, step)):
                    order = np.lexsort((np.arange(len(row)), -row.astype(np.float64)))
                    if row[order[w.m]] - row[order[w.m + 1]] < 32 * T:
                        continue             # x_{m+1} not alone at T -> 0
                    kids = np.nonzero(nb["parent"] == uid)[0]
                    y = [int(nb["token"][c]) for c in kids if nb["kind"][c] == 1]
                    assert y == [int(order[w.m])], (name, step, b, uid)
    assert differs
