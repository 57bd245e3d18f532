"""Whole decoding steps through the C ABI, with the draft / target model
replaced by a row callback.

``run_step`` is the reference sequence of calls: begin_step, expand_level at
every depth (feeding the draft logits of the frontier the library chose),
prune, then verify on the target logits of the pruned tree.  The callbacks
receive node path keys; ``synth`` turns keys into logits for the synthetic
workloads.  Host syncs happen only where a real engine would run its model
(reading the frontier / pruned tree to know which rows to compute).
"""

import torch

import synth
from .binding import Tree


def make_tree(w, device="cuda", **over):
    kw = dict(batch=w.B, vocab=w.V, pool=w.K, leads=w.m, depth=w.depth,
              support=w.support, n_expand=w.n_expand,
              construct_tempered=w.construct_tempered, eps_m0=w.eps_m0, method=w.method,
              construct_full=w.construct_full,
              dtype=torch.bfloat16 if w.dtype == "bf16" else torch.float32,
              device=device)
    kw.update(over)
    return Tree(**kw)


def _rows(w, keys, device, stride):
    rows = synth.draft_rows(w, keys, device=device)
    if stride == w.V:
        return rows
    out = torch.zeros((rows.shape[0], stride), dtype=rows.dtype, device=device)
    out[:, :w.V] = rows
    return out


def _trows(w, keys, sigmas, device, stride):
    rows = synth.target_rows(w, keys, sigmas, device=device)
    if stride == w.V:
        return rows
    out = torch.zeros((rows.shape[0], stride), dtype=rows.dtype, device=device)
    out[:, :w.V] = rows
    return out


def run_step(tree, w, step, T=None, device="cuda", record=None):
    """One step for all sequences of workload ``w``; returns
    (accepted [B, D], accept_len [B], final_token [B]) as CPU tensors.
    ``record`` (a dict) receives the logit buffers fed to the library."""
    T = w.T if T is None else T
    B, NE, V = w.B, w.n_expand, w.V
    stride = tree.row_stride
    key = synth.step_rng_key(w, step)
    keys = [[synth.root_key(w, b, step)] for b in range(B)]
    tree.begin_step()
    drafts = []
    for d in range(w.depth):
        P = len(keys[0])
        flat = [k for ks in keys for k in ks]
        rows = _rows(w, flat, device, stride).view(B, P, stride)
        drafts.append(rows)
        tree.expand_level(rows, T, key)
        if d + 1 < w.depth:
            par, tok = tree.frontier()
            par = par.cpu().tolist()
            tok = tok.cpu().tolist()
            keys = [[synth.child_key(keys[b][par[b][j]], tok[b][j]) for j in range(NE)]
                    for b in range(B)]
    tree.prune(w.R)
    ppar, ptok = tree.pruned_view()
    ppar = ppar.cpu().tolist()
    ptok = ptok.cpu().tolist()
    pkeys = []
    for b in range(B):
        ks = [synth.root_key(w, b, step)]
        for i in range(1, w.R + 1):
            ks.append(synth.child_key(ks[ppar[b][i]], ptok[b][i]))
        pkeys.append(ks)
    flat = [k for ks in pkeys for k in ks]
    sig = [synth.seq_sigma_t(w, b) for b in range(B) for _ in range(w.R + 1)]
    target = _trows(w, flat, sig, device, stride).view(B, w.R + 1, stride)
    acc, alen, fin = tree.verify(target, T, key)
    if record is not None:
        record["draft"] = drafts
        record["target"] = target
        record["rng_key"] = key
        record["T"] = T
    return acc.cpu(), alen.cpu(), fin.cpu()


def replay_step(tree, rec, R, out=None, stream=None):
    """The library calls of one recorded step (no host work in between)."""
    tree.begin_step()
    for rows in rec["draft"]:
        tree.expand_level(rows, rec["T"], rec["rng_key"], stream=stream)
    tree.prune(R, stream=stream)
    return tree.verify(rec["target"], rec["T"], rec["rng_key"], out=out, stream=stream)
