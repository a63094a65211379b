"""Runs oracle functions over many independent inputs on a pool of CPU
processes (test infrastructure; no GPU use in the workers).

The oracle's block quantizers are plain numpy and take seconds per DeepSeek-
V3 expert matrix; the full-size parity tests need tens of expert matrices
and thousands of activation rows, whose quantizations are independent of one
another.  Workers are spawned (fresh interpreters that import numpy and the
oracle only), never forked from a process that uses the GPU.
"""
from __future__ import annotations

import concurrent.futures as cf
import multiprocessing as mp
import os

import numpy as np

import oracle

_POOL = None


def _workers() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def pool():
    global _POOL
    if _POOL is None:
        _POOL = cf.ProcessPoolExecutor(max_workers=_workers(), mp_context=mp.get_context("spawn"))
    return _POOL


def quantize_weights(mats):
    """oracle.quantize_weight over a list of fp32 matrices -> list of (q, s)."""
    return list(pool().map(oracle.quantize_weight, mats))


def quant_act_rows(x_bits: np.ndarray, rows_per_task: int = 256):
    """oracle.quant_act over bf16 rows [T, H], split into independent row blocks."""
    parts = [x_bits[i:i + rows_per_task] for i in range(0, x_bits.shape[0], rows_per_task)]
    res = list(pool().map(oracle.quant_act, parts))
    return np.concatenate([q for q, _ in res]), np.concatenate([s for _, s in res])
