"""rheo_create_static: a tree whose device state lives in the library's
static scratch array (no device allocation) gives the same results, bit
for bit, as a tree from rheo_create -- on two calls in a row on one device,
the second with a smaller input (a dense tree, in the region the first one
used), over two steps each."""

import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2609_21827_amd import binding
    binding.load_library()
    return "cuda"


def _steps(tree, w, steps, dev):
    from paper_2609_21827_amd.driver import run_step
    out = []
    for s in steps:
        acc, alen, fin = run_step(tree, w, s, device=dev)
        nodes = {k: v.cpu().numpy() for k, v in tree.read_nodes().items()}
        pv = [x.cpu().numpy() for x in tree.pruned_view()]
        out.append((acc.numpy(), alen.numpy(), fin.numpy(), nodes, pv))
    torch.cuda.synchronize()
    assert tree.device_error() == 0
    return out


def test_static_tree_matches_allocated_tree(dev):
    from paper_2609_21827_amd.driver import make_tree
    first = W["headline"].with_(name="static_a", B=16, depth=5, R=40)
    second = W["llama2"].with_(name="static_b", B=3, support=0, depth=4, R=20)
    assert second.B * second.V < first.B * first.V
    for w in (first, second):
        ref_tree = make_tree(w, device=dev)
        ref = _steps(ref_tree, w, [0, 1], dev)
        ref_tree.close()
        st = make_tree(w, device=dev, static=True)
        got = _steps(st, w, [0, 1], dev)
        st.close()
        for (a1, l1, f1, n1, p1), (a2, l2, f2, n2, p2) in zip(got, ref):
            assert np.array_equal(a1, a2) and np.array_equal(l1, l2) and np.array_equal(f1, f2)
            for k in n1:
                assert np.array_equal(n1[k], n2[k]), (w.name, k)
            for x, y in zip(p1, p2):
                assert np.array_equal(x, y), w.name
