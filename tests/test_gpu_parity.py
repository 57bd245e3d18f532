"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Both sides see the same seeded synthetic logits (``synth``), generated from
the node path keys each side derives from its *own* tree, so a divergence
anywhere shows up as different rows as well as different records.  The bar
(set by the target): tree topology, token ids, slot kinds, pruned set,
accepted tokens and final tokens bit-exact; probabilities within 1e-5
relative -- they are in fact compared bit-exactly, since both sides evaluate
the same fp32 / integer / correctly rounded fp64 operation sequence.
"""

import os

import numpy as np
import pytest
import torch

import synth
from oracle import rheo
from oracle.harness import node_table, oracle_step

pytestmark = pytest.mark.gpu

INT_FIELDS = ("token", "parent", "depth", "slot", "kind")
FP_FIELDS = ("proxy", "qtrue", "score")


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2609_21827_amd import binding
    binding.load_library()
    return "cuda"


def _check_seq(w, tree_nodes, ppar, ptok, acc, alen, fin, b, step, T, mask=None, depth=None):
    print(f"  oracle {w.name} b={b} step={step} T={T}", flush=True)
    nodes, pt, oacc, ou = oracle_step(w, b, step, T=T)
    tab = node_table(nodes)
    for k in INT_FIELDS:
        got = tree_nodes[k][b]
        assert np.array_equal(got, tab[k]), (k, b, np.nonzero(got != tab[k])[0][:10])
    for k in FP_FIELDS:
        got = tree_nodes[k][b]
        want = tab[k]
        rel = np.abs(got - want) / np.maximum(np.abs(want), 1e-300)
        assert np.all(rel <= 1e-5), (k, b, float(rel.max()))
        assert np.array_equal(got, want), (k, b, float(rel.max()))
    R = len(pt.order) - 1
    assert list(ptok[b][:R + 1]) == [-1] + [nodes[u].token for u in pt.order[1:]]
    assert list(ppar[b][:R + 1]) == list(pt.parent)
    if mask is not None:
        om, od = rheo.tree_mask(nodes, pt)
        assert np.array_equal(mask[b], np.array(om, dtype=np.uint8)), b
        assert list(depth[b]) == od
    n = int(alen[b])
    assert list(acc[b][:n]) == list(oacc), (b, list(acc[b][:n]), oacc)
    assert all(x == -1 for x in acc[b][n:])
    assert int(fin[b]) == ou


def run_parity(w, steps, seqs, T=None, dev="cuda", tree_kw=None, env=None):
    from paper_2609_21827_amd.driver import make_tree, run_step
    T = w.T if T is None else T
    os.environ.update(env or {})
    try:
        tree = make_tree(w, device=dev, **(tree_kw or {}))
    finally:
        for k in env or {}:
            del os.environ[k]
    try:
        for step in steps:
            print(f"gpu step {w.name} step={step} T={T}", flush=True)
            acc, alen, fin = run_step(tree, w, step, T=T, device=dev)
            nodes = {k: v.cpu().numpy() for k, v in tree.read_nodes().items()}
            ppar, ptok = (x.cpu().numpy() for x in tree.pruned_view())
            mask, depth = (x.cpu().numpy() for x in tree.tree_mask())
            torch.cuda.synchronize()
            assert tree.device_error() == 0
            for b in seqs:
                _check_seq(w, nodes, ppar, ptok, acc.numpy(), alen.numpy(), fin.numpy(),
                           b, step, T, mask, depth)
    finally:
        tree.close()


W = synth.WORKLOADS


def test_tiny_many_steps(dev):
    run_parity(W["tiny"], range(120), [0], dev=dev)


@pytest.mark.parametrize("over", [
    dict(m=0), dict(m=2), dict(K=1, m=0, R=3, n_expand=1), dict(depth=1, R=3), dict(R=1), dict(R=21),
    dict(construct_tempered=True, T=0.6), dict(T=2.0), dict(n_expand=2, R=7),
    dict(B=3), dict(eps_m0=2.0 ** -20, m=0),
])
def test_tiny_variants(dev, over):
    w = W["tiny"].with_(**over)
    run_parity(w, range(25), list(range(w.B)), dev=dev)


@pytest.mark.parametrize("over", [
    dict(V=1001, dtype="f32", recipe="zipf", support=128, K=5, depth=4, R=20),
    dict(V=1003, dtype="bf16", recipe="zipf", support=128, K=5, depth=4, R=20),
    # a small support makes the row's last, partial vector matter often
    dict(V=1003, dtype="bf16", recipe="zipf", support=6, K=5, depth=4, R=20, B=3),
    dict(V=200, dtype="bf16", recipe="zipf", support=1024, K=6, depth=3, R=15),
    dict(V=300, dtype="bf16", recipe="flat", support=128, K=4, depth=3, R=12),
    dict(V=5000, dtype="bf16", recipe="zipf", quantum=0.5, support=128, K=4, depth=3, R=12),
    dict(V=32000, dtype="f32", recipe="zipf", support=1024, K=8, depth=3, R=30),
    dict(V=4099, dtype="f32", recipe="zipf_t3", support=64, K=6, depth=5, R=40, B=2),
    dict(V=128256, dtype="bf16", recipe="zipf", support=512, K=8, depth=2, R=10),
    dict(V=70001, dtype="bf16", recipe="zipf", quantum=2.0, support=128, K=4, depth=2, R=6),
    # rows of more than 16384 vectors: 48 vectors per thread in the row kernel
    dict(V=70001, dtype="f32", recipe="zipf", support=128, K=4, depth=2, R=6),
    dict(V=180001, dtype="bf16", recipe="zipf", quantum=1.0, support=256, K=4, depth=2, R=6),
    dict(V=160001, dtype="bf16", recipe="zipf", support=512, K=6, depth=2, R=10),
    # rows too long for the row kernel (more than 24576 vectors): the
    # chunked pair on every level; the largest vocabulary the library takes
    dict(V=100003, dtype="f32", recipe="zipf", support=128, K=4, depth=2, R=6),
    dict(V=262143, dtype="bf16", recipe="zipf", support=256, K=4, depth=2, R=6),
    # supports above 256: the whole row as the support, a support that is
    # no power of two, and massive ties at the threshold
    dict(V=1003, dtype="bf16", recipe="zipf", support=1024, K=5, depth=3, R=12),
    dict(V=300, dtype="f32", recipe="zipf", support=300, K=4, depth=3, R=12),
    dict(V=32000, dtype="bf16", recipe="zipf", quantum=0.5, support=700, K=6, depth=3, R=20),
    # the support's boundary among hundreds of zero logits of both signs
    # (Gaussian logits rounded to multiples of 8: -0.0 below zero)
    dict(V=1003, dtype="bf16", recipe="gauss", quantum=8.0, support=128, K=5, depth=3, R=12),
    dict(V=1003, dtype="f32", recipe="gauss", quantum=8.0, support=128, K=5, depth=3, R=12),
    dict(V=4099, dtype="bf16", recipe="gauss", quantum=8.0, support=300, K=5, depth=3, R=12),
])
@pytest.mark.parametrize("row", ["auto", "0", "narrow"])
def test_edge_shapes(dev, over, row):
    """row "0": every sparse level on the chunked pair; "narrow": the row
    kernel with 256-thread blocks wherever it takes the row."""
    w = W["tiny"].with_(name="edge", sigma=1.5, sigma_t=0.8, **over)
    tree_kw = {}
    if w.V % 8:
        tree_kw["row_stride"] = (w.V + 7) // 8 * 8
    env = {"0": {"RHEO_EXPAND_ROW": "0"}, "narrow": {"RHEO_ROW_NARROW": "1"}}.get(row)
    run_parity(w, range(3), list(range(w.B)), dev=dev, tree_kw=tree_kw, env=env)


def _root_guess_misses(w, steps):
    """Root rows (always verified) whose target maximum lies outside the
    draft's top-S (dense mode: top-K, the children): there the row maximum
    is not at a special token."""
    n = 0
    for step in steps:
        keys = [synth.root_key(w, b, step) for b in range(w.B)]
        d = synth.as_fp32_numpy(synth.draft_rows(w, keys))
        t = synth.as_fp32_numpy(synth.target_rows(
            w, keys, [synth.seq_sigma_t(w, b) for b in range(w.B)]))
        S = min(w.support, w.V) if w.support > 0 else w.K
        for b in range(w.B):
            n += int(t[b].argmax()) not in set(np.argsort(-d[b], kind="stable")[:S].tolist())
    return n


@pytest.mark.parametrize("over", [
    dict(V=1003, dtype="bf16", support=16),
    dict(V=1001, dtype="f32", support=16),
    dict(V=4099, dtype="bf16", support=300),
    # dense mode: the special tokens are the children
    dict(V=1003, dtype="bf16", support=0),
    dict(V=1001, dtype="f32", support=0),
])
def test_verify_row_max_off_special_tokens(dev, over):
    """Target rows far from the draft (sigma_t = 8): the row maximum is
    seldom at a special token, so the verification layer's guess of it
    misses and the maximum is exchanged before the weights are redone."""
    w = W["tiny"].with_(name="guess_miss", recipe="zipf", K=5, depth=3, R=12, B=4,
                        sigma=1.5, sigma_t=8.0, **over)
    assert _root_guess_misses(w, range(4)) >= 8
    run_parity(w, range(4), list(range(w.B)), dev=dev,
               tree_kw={"row_stride": (w.V + 7) // 8 * 8})


def test_verify_row_max_off_special_tokens_llama3(dev):
    w = W["llama3"].with_(name="llama3_guess_miss", sigma_t=6.0, B=2)
    assert _root_guess_misses(w, [0]) == 2
    run_parity(w, [0], [0, 1], dev=dev)


def test_llama2(dev):
    run_parity(W["llama2"], range(3), [0], dev=dev)


@pytest.mark.parametrize("T", [0.6, 1.0])
def test_llama3_sparse(dev, T):
    run_parity(W["llama3"], range(2), [0], T=T, dev=dev)


def test_batched(dev):
    run_parity(W["batched"], [0], [0, 17, 42, 63], dev=dev)


def test_large(dev):
    run_parity(W["large"], [0], [0, 77, 127], dev=dev)


def test_headline(dev):
    run_parity(W["headline"], [0, 1], [0, 31, 63], dev=dev)


def test_headline_all_sequences(dev):
    # every sequence of the batch (every row block of every level), two steps
    run_parity(W["headline"], [20, 21], list(range(64)), dev=dev)


@pytest.mark.parametrize("support", [256, 512, 1024])
def test_headline_supports(dev, support):
    # the larger sparse supports (Sec. 5.5) at the batched shape, where
    # every level runs one block per row
    w = W["headline"].with_(name=f"headline_s{support}", support=support, depth=4, R=30)
    run_parity(w, [0], [0, 63], dev=dev)


def test_support_fallback_rows(dev):
    # sequences 30 and 40 of step 2 at support 256 each hold a row whose
    # candidates overflow LDS (exact re-selection from the row), once
    # miscounted after the out-of-line fallback
    w = W["headline"].with_(name="headline_s256", support=256)
    run_parity(w, [2], [30, 40], dev=dev)


# ---- whole-vocabulary construction with a sparse tail (Sec. 5.5 reading)
@pytest.mark.parametrize("over", [dict(support=16), dict(support=16, construct_tempered=True, T=0.6),
                                  dict(support=8, m=0, K=4, R=10)])
def test_construct_full_tiny(dev, over):
    w = W["tiny"].with_(name="tiny_full", construct_full=True, **over)
    run_parity(w, range(30), [0], dev=dev)


def test_construct_full_llama2(dev):
    run_parity(W["llama2"].with_(name="llama2_full", construct_full=True), range(2), [0], dev=dev)


@pytest.mark.parametrize("support,row", [(128, "auto"), (128, "0"), (512, "auto")])
def test_construct_full_headline(dev, support, row):
    w = W["headline"].with_(name="headline_full", construct_full=True, support=support,
                            depth=3, R=20)
    env = {"RHEO_EXPAND_ROW": row} if row != "auto" else None
    run_parity(w, [0], [0, 63], dev=dev, env=env)


SHAPES = (
    {},
    {"RHEO_EXPAND_VARIANT": "0", "RHEO_VERIFY_BLOCKS": "4"},
    {"RHEO_EXPAND_VARIANT": "3", "RHEO_VERIFY_BLOCKS": "64"},
    {"RHEO_EXPAND_VARIANT": "1", "RHEO_VERIFY_BLOCKS": "1024"},
    {"RHEO_EXPAND_ROW": "1"},
    {"RHEO_EXPAND_ROW": "0", "RHEO_VERIFY_BLOCKS": "256"},
    {"RHEO_ROW_NARROW": "1"},
    {"RHEO_ROW_NARROW": "0"},
)


@pytest.mark.parametrize("wl", ["llama3", "llama2", "quantum_bf16"])
def test_launch_shape_independence(dev, wl):
    """Results do not depend on the expand kernels (chunk size, one block per
    row) or the verification team size."""
    from paper_2609_21827_amd.driver import make_tree, run_step
    if wl == "llama3":
        w = W["llama3"].with_(B=4)
    elif wl == "llama2":
        w = W["llama2"].with_(B=2, depth=4, R=30)
    else:   # massive ties: the exact fallbacks of both selection kernels
        w = W["llama3"].with_(name="quantum_bf16", B=2, depth=3, R=20, recipe="zipf",
                              quantum=2.0)
    outs = []
    for env in SHAPES:
        os.environ.update(env)
        try:
            tree = make_tree(w, device=dev)
        finally:
            for k in env:
                del os.environ[k]
        acc, alen, fin = run_step(tree, w, 0, device=dev)
        nodes = tree.read_nodes()
        outs.append((acc, alen, fin, {k: v.cpu() for k, v in nodes.items()}))
        assert tree.device_error() == 0
        tree.close()
    for o in outs[1:]:
        assert torch.equal(o[0], outs[0][0]) and torch.equal(o[1], outs[0][1])
        assert torch.equal(o[2], outs[0][2])
        for k in o[3]:
            assert torch.equal(o[3][k], outs[0][3][k]), k


def test_step_order_enforced(dev):
    from paper_2609_21827_amd.binding import RheoError, RHEO_ESTATE
    from paper_2609_21827_amd.driver import make_tree
    w = W["tiny"]
    tree = make_tree(w, device=dev)
    rows = torch.zeros((1, 1, w.V), dtype=torch.float32, device=dev)
    with pytest.raises(RheoError) as e:
        tree.expand_level(rows, 1.0, 1)
    assert e.value.code == RHEO_ESTATE
    tree.begin_step()
    with pytest.raises(RheoError):
        tree.prune(3)
    with pytest.raises(RheoError):
        tree.expand_level(rows, 0.0, 1)
    tree.close()


@pytest.mark.parametrize("support", [128, 0])
def test_step_args_fixed(dev, support):
    """T and rng_key are the step's: a later expand level or the verify call
    with another value is refused before anything is enqueued."""
    from paper_2609_21827_amd.binding import RheoError, RHEO_EINVAL
    from paper_2609_21827_amd.driver import make_tree
    w = W["tiny"].with_(support=support)
    tree = make_tree(w, device=dev)
    dt = torch.float32
    tree.begin_step()
    tree.expand_level(torch.zeros((1, 1, w.V), dtype=dt, device=dev), 1.0, 5)
    rows = torch.zeros((1, w.n_expand, w.V), dtype=dt, device=dev)
    for T, key in ((0.9, 5), (1.0, 6)):
        with pytest.raises(RheoError) as e:
            tree.expand_level(rows, T, key)
        assert e.value.code == RHEO_EINVAL
    for _ in range(w.depth - 1):
        tree.expand_level(rows, 1.0, 5)
    tree.prune(w.R)
    target = torch.zeros((1, w.R + 1, w.V), dtype=dt, device=dev)
    for T, key in ((0.9, 5), (1.0, 6)):
        with pytest.raises(RheoError) as e:
            tree.verify(target, T, key)
        assert e.value.code == RHEO_EINVAL
    acc, alen, fin = tree.verify(target, 1.0, 5)
    torch.cuda.synchronize()
    assert int(alen[0]) >= 0 and tree.device_error() == 0
    tree.close()


def test_verify_timeout_failure_then_recovery(dev):
    """A team wait that gives up (forced from the host with a zero spin
    limit) ends each affected walk with the failure result, never a silent
    partial walk; the next call on the same handle, whose team words still
    hold the failed call's values, is exact again."""
    from paper_2609_21827_amd.driver import make_tree, replay_step, run_step
    w = W["headline"].with_(name="spin", B=16, depth=3, R=20)
    tree = make_tree(w, device=dev)
    rec = {}
    ref = run_step(tree, w, 0, device=dev, record=rec)
    torch.cuda.synchronize()
    assert tree.device_error() == 0
    os.environ["RHEO_VERIFY_SPIN"] = "0"
    try:
        out = [x.cpu() for x in replay_step(tree, rec, w.R)]
    finally:
        del os.environ["RHEO_VERIFY_SPIN"]
    assert tree.device_error() & 128
    failed = 0
    for b in range(w.B):
        if int(out[1][b]) == -1:
            failed += 1
            assert int(out[2][b]) == -1 and bool((out[0][b] == -1).all()), b
        else:               # the team's first block saw every exchange complete
            assert all(torch.equal(o[b], r[b]) for o, r in zip(out, ref)), b
    assert failed > 0
    again = [x.cpu() for x in replay_step(tree, rec, w.R)]
    for o, r in zip(again, ref):
        assert torch.equal(o, r)
    tree.close()


def test_generator_cpu_gpu_identical(dev):
    for name in ("llama2", "large", "tiny"):
        w = W[name]
        keys = [synth.root_key(w, b, 3) for b in range(3)]
        a = synth.draft_rows(w, keys, device="cpu")
        g = synth.draft_rows(w, keys, device=dev).cpu()
        assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a,
                           g.view(torch.int16) if g.dtype == torch.bfloat16 else g)
        ta = synth.target_rows(w, keys, [0.9] * 3, device="cpu")
        tg = synth.target_rows(w, keys, [0.9] * 3, device=dev).cpu()
        assert torch.equal(ta.float(), tg.float())


def test_frontier_view_matches_copy(dev):
    """The zero-copy frontier view and rheo_frontier's copy agree at every
    level, and match the oracle's frontier (via the step's parity above)."""
    from paper_2609_21827_amd.driver import make_tree
    import synth
    w = W["llama2"].with_(B=3, depth=4, R=30)
    tree = make_tree(w, device=dev)
    view = tree.frontier_view()
    keys = [[synth.root_key(w, b, 0)] for b in range(w.B)]
    tree.begin_step()
    for d in range(w.depth):
        P = len(keys[0])
        flat = [k for ks in keys for k in ks]
        rows = synth.draft_rows(w, flat, device=dev).view(w.B, P, w.V)
        tree.expand_level(rows, w.T, synth.step_rng_key(w, 0))
        if d + 1 < w.depth:
            par, tok = tree.frontier()
            torch.cuda.synchronize()
            assert torch.equal(par, view[0]) and torch.equal(tok, view[1])
            p, t = par.cpu().tolist(), tok.cpu().tolist()
            keys = [[synth.child_key(keys[b][p[b][j]], t[b][j]) for j in range(w.n_expand)]
                    for b in range(w.B)]
    assert tree.device_error() == 0
    tree.close()


@pytest.mark.parametrize("support", [128, 0])
@pytest.mark.parametrize("between", [True, False])
def test_graph_replay_matches_eager(dev, support, between):
    """A captured step replays bit-exactly, several times: with eager steps
    and synchronisations between the replays, and back to back (the
    verification teams' barrier words then hold the previous replay's
    values; the dense walk's team barriers once took those for current)."""
    from paper_2609_21827_amd.driver import make_tree, run_step
    w = W["llama3"].with_(B=3, depth=4, R=20, support=support)
    tree = make_tree(w, device=dev)
    rec = {}
    acc, alen, fin = run_step(tree, w, 0, device=dev, record=rec)
    ref = (acc.cpu(), alen.cpu(), fin.cpu())
    out = tuple(torch.empty_like(x, device=dev) for x in (acc, alen, fin))
    pv = tuple(torch.empty((w.B, w.R + 1), dtype=torch.int32, device=dev) for _ in range(2))
    cap = torch.cuda.Stream()

    def step(stream):
        tree.begin_step()
        for rows in rec["draft"]:
            tree.expand_level(rows, rec["T"], rec["rng_key"], stream=stream)
        tree.prune(w.R, stream=stream)
        tree.pruned_view(out=pv, stream=stream)
        tree.verify(rec["target"], rec["T"], rec["rng_key"], out=out, stream=stream)

    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=cap):
        step(cap)
    torch.cuda.synchronize()
    for r in range(4):
        for o in out:
            o.fill_(-5)
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(out, ref):
            assert torch.equal(a.cpu(), b), f"replay {r}"
        if between:
            run_step(tree, w, 1 + r, device=dev)      # eager work in between
            torch.cuda.synchronize()
    assert tree.device_error() == 0
    tree.close()


# ---- dense mode: the support is the whole vocabulary ---------------------

def test_dense_tiny_many_steps(dev):
    run_parity(W["tiny"].with_(name="tiny_dense", support=0), range(60), [0], dev=dev)


@pytest.mark.parametrize("over", [
    dict(), dict(K=1, m=0, R=3, n_expand=1), dict(m=0, eps_m0=2.0 ** -20),
    dict(construct_tempered=True, T=0.6), dict(T=2.0), dict(B=3), dict(K=4, m=2, R=10),
])
def test_dense_tiny_variants(dev, over):
    w = W["tiny"].with_(name="tiny_dense", support=0, **over)
    run_parity(w, range(12), list(range(w.B)), dev=dev)


@pytest.mark.parametrize("over", [
    dict(V=1001, dtype="f32", recipe="zipf", K=5, depth=4, R=20),
    dict(V=1003, dtype="bf16", recipe="zipf", K=5, depth=4, R=20),
    dict(V=300, dtype="bf16", recipe="flat", K=4, depth=3, R=12),
    dict(V=5000, dtype="bf16", recipe="zipf", quantum=0.5, K=4, depth=3, R=12),
    dict(V=4099, dtype="f32", recipe="zipf_t3", K=6, depth=4, R=30, B=2, T=0.6),
    dict(V=70001, dtype="bf16", recipe="zipf", K=8, depth=2, R=10),
])
def test_dense_edge_shapes(dev, over):
    w = W["tiny"].with_(name="edge_dense", sigma=1.5, sigma_t=0.8, support=0, **over)
    tree_kw = {}
    if w.V % 8:
        tree_kw["row_stride"] = (w.V + 7) // 8 * 8
    run_parity(w, range(2), list(range(w.B)), dev=dev, tree_kw=tree_kw)


@pytest.mark.parametrize("support", [0, 16])
def test_near_ties(dev, support):
    """Distinct logits a few ulps below the maximum share its integer weight:
    ranks by (weight, id) then differ from ranks by logit (dense mode takes
    its exact fallbacks; sparse mode its tie-aware ranking)."""
    w = W["tiny"].with_(name="near_ties", V=1001, dtype="f32", recipe="zipf", sigma=1.5,
                        sigma_t=0.8, K=3, m=1, depth=3, R=8, support=support, near_ties=6)
    run_parity(w, range(4), [0], dev=dev, tree_kw={"row_stride": 1004})


def test_dense_llama2(dev):
    run_parity(W["llama2"].with_(name="llama2_dense", support=0, depth=4, R=30), range(2), [0],
               dev=dev)


def test_dense_llama3(dev):
    run_parity(W["llama3"].with_(name="llama3_dense", support=0, depth=3, R=20), [0], [0],
               T=0.6, dev=dev)


def test_dense_batched(dev):
    w = W["headline"].with_(name="headline_dense", support=0, B=8, depth=3, R=20)
    run_parity(w, [0], [0, 5], dev=dev)


def test_headline_dense(dev):
    """The dense bench workload at its full size, sampled sequences."""
    run_parity(W["headline_dense"], [0], [0, 63], dev=dev)


# ---- the comparison methods: RRSw verification, pure top-K trees ----------

METHOD_OVERS = [dict(), dict(m=2, K=4, R=10), dict(m=0, eps_m0=2.0 ** -20),
                dict(T=0.6, construct_tempered=True), dict(B=3)]


@pytest.mark.parametrize("method", ["rrsw", "topk"])
@pytest.mark.parametrize("over", METHOD_OVERS)
def test_methods_tiny(dev, method, over):
    w = W["tiny"].with_(name="tiny_" + method, method=method, **over)
    run_parity(w, range(30), list(range(w.B)), dev=dev)


@pytest.mark.parametrize("method", ["rrsw", "topk"])
def test_methods_dense_tiny(dev, method):
    w = W["tiny"].with_(name="tiny_dense_" + method, support=0, method=method, m=2, K=4, R=10)
    run_parity(w, range(20), [0], dev=dev)


@pytest.mark.parametrize("method", ["rrsw", "topk"])
def test_methods_llama2_both_modes(dev, method):
    for support in (128, 0):
        w = W["llama2"].with_(name="llama2_" + method, method=method, support=support,
                              m=2, depth=3, R=20)
        run_parity(w, range(2), [0], dev=dev)


@pytest.mark.parametrize("method", ["rrsw", "topk"])
def test_methods_headline(dev, method):
    """The batched bench shape (one block per row at every level)."""
    run_parity(W["headline"].with_(name="headline_" + method, method=method), [0], [0, 63],
               dev=dev)


@pytest.mark.parametrize("method,over", [
    ("rrsw", dict(support=512, depth=3, R=20)),                  # large-support pools
    ("topk", dict(support=1024, depth=3, R=20)),
    ("rrsw", dict(construct_full=True, depth=3, R=20)),          # whole-vocabulary q
    ("topk", dict(construct_full=True, support=256, depth=3, R=20)),
    ("rrsw", dict(support=0, B=8, depth=3, R=20)),               # dense, batched shape
    ("topk", dict(support=0, B=8, depth=3, R=20)),
])
def test_method_combinations(dev, method, over):
    w = W["headline"].with_(name=f"headline_{method}_combo", method=method, **over)
    run_parity(w, [0], [0, w.B - 1], dev=dev)


def _many_steps(w, steps, dev):
    """Steps in a row on one handle, the device error flag after each, and
    one sequence of each step against the oracle."""
    from paper_2609_21827_amd.driver import make_tree, run_step
    tree = make_tree(w, device=dev)
    try:
        for step in steps:
            print(f"gpu step {w.name} step={step}", flush=True)
            acc, alen, fin = run_step(tree, w, step, device=dev)
            nodes = {k: v.cpu().numpy() for k, v in tree.read_nodes().items()}
            ppar, ptok = (x.cpu().numpy() for x in tree.pruned_view())
            torch.cuda.synchronize()
            assert tree.device_error() == 0, step
            b = (13 * step + 5) % w.B
            _check_seq(w, nodes, ppar, ptok, acc.numpy(), alen.numpy(), fin.numpy(), b, step, w.T)
    finally:
        tree.close()


def test_headline_many_steps(dev):
    _many_steps(W["headline"], range(2, 12), dev)


@pytest.mark.parametrize("support", [256, 1024])
def test_large_supports_many_steps(dev, support):
    w = W["headline"].with_(name=f"headline_s{support}", support=support)
    _many_steps(w, range(3, 9), dev)
