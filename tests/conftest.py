import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def gpu_available() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


def oracle_score_threaded(C, H, bits, G, chunk: int = 1024, workers: int = 0):
    """oracle.score over row chunks on a thread pool (numpy releases the GIL
    in its array kernels); the same rows, arithmetic and order as
    oracle.score, only spread over the host cores."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle
    n = C.shape[0]
    if workers <= 0:
        workers = max(1, min(16, os.cpu_count() or 1))
    starts = list(range(0, n, chunk))
    try:  # one BLAS thread per worker: the pool already uses every core
        from threadpoolctl import threadpool_limits
        limit = threadpool_limits(1)
    except Exception:  # pragma: no cover
        limit = None
    try:
        with ThreadPoolExecutor(workers) as ex:
            parts = list(ex.map(lambda i: oracle.score_rows(C[i:i + chunk], H, bits, G), starts))
    finally:
        if limit is not None:
            limit.restore_original_limits()
    return np.concatenate(parts, axis=0) if parts else np.zeros((0, len(bits)))
