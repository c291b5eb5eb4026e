"""Run the oracle over many sentences in parallel host processes.

Test infrastructure: each worker process builds the same seeded model once
(synth.generate is deterministic) and runs the unchanged oracle on one
sentence per task.  Workers are started with the "spawn" method, so none of
them inherits the parent's GPU state.
"""
from __future__ import annotations

import concurrent.futures as cf
import multiprocessing as mp
import os

import numpy as np

_model = None


def _init(cfg):
    global _model
    import oracle
    from synth import generate as G

    _model = oracle.Model(G.build_model(cfg))


def _beam_one(args):
    src_row, n, W, steps, alpha = args
    out, out_len, score = _model.beam(src_row[None, :], np.array([n], np.int32), W, steps, alpha)
    return out[0], int(out_len[0]), score[0]


def beam_many(cfg, src, lens, idx, W, steps, alpha, workers: int = 16):
    """Oracle beam search of sentences idx of (src, lens): (out [k, steps],
    out_len [k], score [k]) in the order of idx."""
    idx = list(idx)
    n_proc = max(1, min(workers, os.cpu_count() or 1, len(idx)))
    tasks = [(np.ascontiguousarray(src[i, : lens[i]]), int(lens[i]), W, steps, alpha) for i in idx]
    with cf.ProcessPoolExecutor(n_proc, mp_context=mp.get_context("spawn"), initializer=_init,
                                initargs=(cfg,)) as ex:
        res = list(ex.map(_beam_one, tasks))
    return (np.stack([r[0] for r in res]), np.array([r[1] for r in res], np.int32),
            np.array([r[2] for r in res], np.float32))
