"""Runs the float64 oracle's per-level recurrent forms over several heads in parallel worker
processes (one head per task, one BLAS thread per worker), for the full-length parity tests whose
oracle would otherwise take minutes in one process.  Test infrastructure only."""

import os
from concurrent.futures import ProcessPoolExecutor
import multiprocessing as mp


def _init_worker():
    from threadpoolctl import threadpool_limits
    threadpool_limits(1)


def _mamba2_head(args):
    from oracle import mamba2
    return mamba2.recurrent(*args)


def _gdn_head(args):
    from oracle import gdn
    return gdn.recurrent(*args)


def recurrent_heads(kind, x, heads, names, workers=None):
    """The oracle's recurrent form ("mamba2" or "gdn") for each (b, h) in `heads`, computed in
    parallel; returns a list of [1, T, 1, d_v] float64 arrays in the order of `heads`."""
    fn = {"mamba2": _mamba2_head, "gdn": _gdn_head}[kind]
    tasks = [tuple(x[n][b:b + 1, :, h:h + 1] for n in names) for b, h in heads]
    n = workers or min(len(tasks), max(1, (os.cpu_count() or 1)), 16)
    with ProcessPoolExecutor(max_workers=n, mp_context=mp.get_context("spawn"), initializer=_init_worker) as ex:
        return list(ex.map(fn, tasks))
