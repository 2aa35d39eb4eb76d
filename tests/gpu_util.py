"""Shared helpers of the GPU tests (test infrastructure only)."""
from __future__ import annotations

import sys

import numpy as np
import torch

from paper_2607_01817_amd import inputs

# The attention tolerance against the fp64 oracle (bf16 operands,
# fp32 accumulation).
MAX_ABS = 2e-2

_cache: dict = {}


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def workload_inputs(name: str, planted: bool = False):
    """Host [S][H][d] tensors of a workload, memoised for the larger ones."""
    key = (name, planted)
    if key not in _cache:
        if len(_cache) >= 2:
            _cache.clear()
        _cache[key] = inputs.make_qkv(inputs.WORKLOADS[name], planted=planted)
    return _cache[key]


def bits(t: torch.Tensor) -> torch.Tensor:
    """Integer view of a tensor's bits (for bit-exact comparison)."""
    t = t.contiguous()
    return t.view(torch.int16) if t.element_size() == 2 else t.view(torch.int32)


def head_major_np(x: torch.Tensor, h: int) -> np.ndarray:
    """Head h of a host [S][H][d] tensor as a float64 [S][d] array."""
    return x[:, h, :].to(torch.float64).numpy()


def check_attention_rows(got_hm: np.ndarray, want: np.ndarray, what: str):
    """got/want: [n][d] float64 rows.  Returns (max_abs, max_abs / max|want|)."""
    err = np.abs(got_hm - want)
    max_abs = float(err.max()) if err.size else 0.0
    ref = float(np.abs(want).max()) if want.size else 0.0
    rel = max_abs / ref if ref > 0 else max_abs
    assert np.all(np.isfinite(got_hm)), f"{what}: non-finite output"
    assert max_abs <= MAX_ABS, f"{what}: max-abs error {max_abs:.3e} > {MAX_ABS}"
    assert rel <= MAX_ABS, f"{what}: normalised error {rel:.3e} > {MAX_ABS} (max|O| = {ref:.3e})"
    return max_abs, rel
