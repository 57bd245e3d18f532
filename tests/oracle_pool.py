"""The oracle's results for many (sequence, step) pairs, computed in worker
processes (CPU only; the workers never touch the GPU).  Used by the GPU
parity tests to check whole batches: each pair is one independent call of
``oracle.harness.oracle_step``.
"""

import multiprocessing as mp
import os
from concurrent.futures import ProcessPoolExecutor

import numpy as np


def _one(job):
    w, b, step, T = job
    import synth
    from oracle import rheo
    from oracle.harness import node_key, node_table, oracle_step
    nodes, pt, acc, u = oracle_step(w, b, step, T=T)
    mask, depth = rheo.tree_mask(nodes, pt)
    root = synth.root_key(w, b, step)
    expanded = [node_key(nodes, n.uid, root) for n in nodes if n.expanded]
    return (b, step), dict(
        tab=node_table(nodes),
        ptok=[-1] + [nodes[x].token for x in pt.order[1:]],
        ppar=list(pt.parent),
        mask=np.array(mask, dtype=np.uint8),
        depth=list(depth),
        acc=list(acc),
        u=int(u),
        expanded_keys=expanded,
    )


def _init_worker():
    # one thread per worker: the pool already uses every core
    import torch
    torch.set_num_threads(1)


def _chunk(jobs):
    return [_one(j) for j in jobs]


def workers():
    """Worker processes: the host's cores, at most 16."""
    return max(1, min(16, os.cpu_count() or 1))


class OraclePool:
    """Submit (w, b, step, T) jobs at once; collect them later (so the
    oracle runs while the GPU works)."""

    def __init__(self, jobs, per_task=1):
        self.ex = ProcessPoolExecutor(max_workers=workers(),
                                      mp_context=mp.get_context("spawn"),
                                      initializer=_init_worker)
        chunks = [jobs[i:i + per_task] for i in range(0, len(jobs), per_task)]
        self.futs = [self.ex.submit(_chunk, c) for c in chunks]

    def results(self):
        out = {}
        try:
            for f in self.futs:
                for k, v in f.result():
                    out[k] = v
        finally:
            self.ex.shutdown()
        return out
