"""The oracle's exact column energies for large inputs, computed on column
blocks in worker processes.

Column j's energy depends on column j alone, so applying the oracle's
``column_energies`` to blocks of columns and concatenating gives exactly its
result on the whole matrix; the workers only spread that work over the
host's cores (spawned processes: they start fresh and never touch the GPU).
The pool must be started before the process first touches the GPU (see
``start``), so that no worker is ever forked from a process holding the
device.  Test infrastructure only."""
from __future__ import annotations

import multiprocessing as mp
import os
import time
from concurrent.futures import ProcessPoolExecutor

import numpy as np

from oracle import rmm_oracle as ro

_POOL = None
# the box gives one GPU job 16 host cores, whatever os.cpu_count() reports
_WORKERS = max(1, min(16, os.cpu_count() or 1))
_SERIAL_BELOW = 1 << 24          # elements; smaller inputs are not worth the hand-off


def start():
    """Start every worker now (call before any GPU use in this process)."""
    global _POOL
    if _POOL is None and _WORKERS > 1:
        _POOL = ProcessPoolExecutor(max_workers=_WORKERS, mp_context=mp.get_context("spawn"))
        # one task per worker: each submit starts a process while none is idle
        list(_POOL.map(time.sleep, [0.5] * _WORKERS))


def stop():
    global _POOL
    if _POOL is not None:
        _POOL.shutdown(wait=True, cancel_futures=True)
        _POOL = None


def _block(A):
    return ro.column_energies(A)


def _block_bf16(bits):
    import workloads as wl
    return ro.column_energies(wl.decode(bits, "bf16"))


def column_energies(A: np.ndarray, bf16_bits: bool = False) -> np.ndarray:
    """ro.column_energies(A) for a 2-D A of float32/float64 values, or of
    bf16 bit patterns (uint16) with ``bf16_bits`` (decoded in the workers)."""
    A = np.asarray(A)
    if A.size < _SERIAL_BELOW or _POOL is None:
        if bf16_bits:
            return _block_bf16(A)
        return ro.column_energies(A)
    K = A.shape[1]
    step = max(1, -(-K // (4 * _WORKERS)))
    parts = [np.ascontiguousarray(A[:, j:j + step]) for j in range(0, K, step)]
    return np.concatenate(list(_POOL.map(_block_bf16 if bf16_bits else _block, parts)))
