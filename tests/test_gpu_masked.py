"""GPU parity on masked vocabularies: logits of -inf (the truncation of
Sec. 3.2; padded vocabularies; constrained decoding), in both dtypes, on
every expand path (chunked, one block per row, large supports, dense), with
masks shared by draft and target and masks of the target alone; rows with
fewer finite logits than the support (the support ends with masked tokens
in id order); and the undefined cases, which set device error bit 9 (512).
The bar is the one of the other parity tests: bit-exact.
"""

import numpy as np
import pytest
import torch

import synth
from test_gpu_configs import run_all
from test_gpu_parity import run_parity

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2609_21827_amd import binding
    binding.load_library()
    return "cuda"


@pytest.mark.parametrize("over", [
    # fewer finite logits than the support (about 100 of 128, 50 of 128)
    dict(V=1003, dtype="bf16", support=128, mask=0.9),
    dict(V=1001, dtype="f32", support=128, mask=0.95),
    # a small support, target-only masks too, three sequences
    dict(V=1003, dtype="bf16", support=6, mask=0.5, mask_target=0.1, B=3),
    # a large support (sorted tail) with about 120 finite of 300
    dict(V=4099, dtype="bf16", support=300, mask=0.97),
    # a padded vocabulary: the last 500 ids masked in every row
    dict(V=1003, dtype="bf16", support=128, mask_tail=500),
    # the support is the whole row, half of it masked
    dict(V=300, dtype="bf16", support=1024, mask=0.5, K=6),
    # leads: none, two
    dict(V=1003, dtype="bf16", support=64, mask=0.8, m=0, mask_target=0.2),
    dict(V=1003, dtype="f32", support=64, mask=0.8, m=2, K=6),
    # dense distributions (support = V)
    dict(V=1003, dtype="bf16", support=0, mask=0.9),
    dict(V=1001, dtype="f32", support=0, mask=0.5, mask_target=0.2),
])
@pytest.mark.parametrize("row", ["auto", "0"])
def test_masked_edge_shapes(dev, over, row):
    kw = dict(recipe="zipf", K=5, depth=3, R=12, sigma=1.5, sigma_t=0.8)
    kw.update(over)
    w = W["tiny"].with_(name="masked_edge", **kw)
    tree_kw = {}
    if w.V % 8:
        tree_kw["row_stride"] = (w.V + 7) // 8 * 8
    env = {"RHEO_EXPAND_ROW": row} if row != "auto" else None
    run_parity(w, range(3), list(range(w.B)), dev=dev, tree_kw=tree_kw, env=env)


@pytest.mark.parametrize("base,over", [
    ("llama2", dict(mask=0.5, mask_target=0.05)),
    ("llama2", dict(mask=0.999)),                 # about 32 finite logits, S = 128
    ("llama3", dict(mask=0.5, mask_target=0.05)),
    ("llama3", dict(mask=0.999)),                 # about 128 finite, around S
    ("llama3", dict(mask_tail=256)),
    ("llama2", dict(mask=0.9, support=0)),
])
def test_masked_workloads(dev, base, over):
    w = W[base].with_(name=base + "_masked", **over)
    run_parity(w, range(2), [0], dev=dev)


@pytest.mark.parametrize("over", [
    dict(mask=0.9, mask_target=0.02),
    dict(mask=0.999),                             # rows below S finite: exact fallback
])
def test_masked_headline_all_sequences(dev, over):
    # the batched shape: one block per row on every level
    run_all(W["headline"].with_(name="headline_masked", **over), [0], dev)


def test_masked_headline_dense(dev):
    run_all(W["headline_dense"].with_(name="headline_dense_masked", mask=0.5, B=16), [0], dev)


def test_undefined_rows_set_error_bit(dev):
    """A draft row whose x_{m+1} is masked, and a target row without a finite
    logit, set device error bit 9; a walk that reaches such a target row
    ends with the failure result; the other sequences are unaffected."""
    from paper_2609_21827_amd.driver import make_tree, replay_step, run_step
    w = W["headline"].with_(name="undef", B=8, depth=3, R=20)
    tree = make_tree(w, device=dev)
    rec = {}
    ref = run_step(tree, w, 0, device=dev, record=rec)
    torch.cuda.synchronize()
    assert tree.device_error() == 0
    # the root target row of sequence 3: all -inf (every walk starts there)
    target = rec["target"].clone()
    target[3, 0, :] = float("-inf")
    out = [x.cpu() for x in replay_step(tree, dict(rec, target=target), w.R)]
    assert tree.device_error() == 512
    assert int(out[1][3]) == -1 and int(out[2][3]) == -1 and bool((out[0][3] == -1).all())
    for b in range(w.B):
        if b != 3:
            assert all(torch.equal(o[b], r[b]) for o, r in zip(out, ref)), b
    tree.close()
    # sequence 5's root draft row with m = 1 finite logit: x_2 is -inf
    tree = make_tree(w, device=dev)
    draft = [d.clone() for d in rec["draft"]]
    keep = int(torch.argmax(draft[0][5, 0, :w.V].float()))
    v = draft[0][5, 0, keep].clone()
    draft[0][5, 0, :] = float("-inf")
    draft[0][5, 0, keep] = v
    out = [x.cpu() for x in replay_step(tree, dict(rec, draft=draft), w.R)]
    assert tree.device_error() & 512
    for b in range(w.B):
        if b != 5:
            assert all(torch.equal(o[b], r[b]) for o, r in zip(out, ref)), b
    tree.close()
