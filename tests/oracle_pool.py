"""Test infrastructure: the oracle's per-cell evaluation and training step run
in a pool of CPU worker processes, for the full-size parity tests whose
oracle work (tens of TFLOP in fp64) is too slow for one process.

The workers are started with "spawn" and import only numpy and the oracle
(never torch or the HIP library), each with one BLAS thread.  The parent
writes the workload, the dataset and the state to a directory; every worker
maps them read-only (copy-on-write for the state, so a training step changes
only the worker's private copy of its unit's row)."""
import json
import multiprocessing as mp
import os

import numpy as np

from oracle import coevo

_W = {}


def _init(path):
    with open(os.path.join(path, "wl.json")) as f:
        wl = json.load(f)
    data = np.load(os.path.join(path, "data.npy"), mmap_mode="r")
    st = coevo.State(**{k: np.load(os.path.join(path, k + ".npy"), mmap_mode="c") for k in coevo.State.FIELDS})
    _W.update(S=coevo.Setup(wl, len(data)), data=data, st=st)


def _eval(args):
    gen, c = args
    L, Lg = coevo.evaluate_cell(_W["S"], _W["st"], _W["data"], gen, c)
    return c, L, Lg


def _train(args):
    gen, step, c = args
    st = _W["st"]
    losses = coevo.train_unit(_W["S"], st, _W["data"], gen, step, c)
    return c, losses, {k: np.array(getattr(st, k)[c]) for k in coevo.State.FIELDS if k != "w"}


class OraclePool:
    """with OraclePool(wl, data, st, tmpdir) as pool: pool.evaluate(gen) / pool.train_step(gen, step)."""

    def __init__(self, wl, data, st, tmpdir, workers=None):
        self.S = coevo.Setup(wl, len(data))
        self.st = st
        path = str(tmpdir)
        with open(os.path.join(path, "wl.json"), "w") as f:
            json.dump(wl, f)
        np.save(os.path.join(path, "data.npy"), np.ascontiguousarray(data))
        for k in coevo.State.FIELDS:
            np.save(os.path.join(path, k + ".npy"), np.ascontiguousarray(getattr(st, k)))
        n = workers or min(16, len(os.sched_getaffinity(0)), self.S.U)
        saved = {k: os.environ.get(k) for k in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")}
        for k in saved:
            os.environ[k] = "1"
        try:
            self.pool = mp.get_context("spawn").Pool(n, initializer=_init, initargs=(path,))
        finally:
            for k, v in saved.items():
                if v is None:
                    os.environ.pop(k, None)
                else:
                    os.environ[k] = v

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.pool.terminate()
        self.pool.join()

    def evaluate(self, gen):
        """(L, Lg, fit_g, fit_d) of every cell, as coevo.evaluate."""
        S = self.S
        L = np.zeros((S.C, S.n, S.n))
        Lg = np.zeros((S.C, S.n, S.n))
        for c, a, b in self.pool.imap_unordered(_eval, [(gen, c) for c in range(S.C)]):
            L[c], Lg[c] = a, b
        fit_d = L.mean(axis=1)
        fit_g = -L.mean(axis=2) if S.wl["fitness_mode"] == 0 else Lg.mean(axis=2)
        return L, Lg, fit_g, fit_d

    def train_step(self, gen, step):
        """coevo.train_step from the pool's state: (losses [U, 2], the new state)."""
        S = self.S
        new = self.st.copy()
        losses = np.zeros((S.U, 2))
        for c, lo, rows in self.pool.imap_unordered(_train, [(gen, step, c) for c in range(S.U)]):
            losses[c] = lo
            for k, v in rows.items():
                getattr(new, k)[c] = v
        return losses, new
