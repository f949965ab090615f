"""Helpers for the GPU parity tests: run the HIP path, compare with the oracle."""
from __future__ import annotations

import sys

import numpy as np

# Tolerances (bf16 inputs, fp32 accumulation; fp32 inputs)
TOL_BF16 = dict(out=5e-3, lse=1e-3, grad=1e-2)
TOL_F32 = dict(out=1e-5, lse=1e-5, grad=1e-5)


def tol(cfg):
    return TOL_BF16 if cfg.dtype == "bf16" else TOL_F32


def announce(msg: str) -> None:
    """Name the case before each GPU step (flushed, so a fault still names it)."""
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


def rel_l2(x, ref) -> float:
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(x - ref) / (den if den > 0 else 1.0))


def lse_err(x, ref) -> float:
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    fin = np.isfinite(ref)
    assert np.array_equal(np.isfinite(x), fin), "lse finiteness pattern differs"
    assert np.all(x[~fin] == ref[~fin]), "lse infinities differ in sign"
    return float(np.max(np.abs(x[fin] - ref[fin]))) if fin.any() else 0.0


def host(t) -> np.ndarray:
    import torch
    t = t.detach()
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.cpu().numpy().astype(np.float64)


def oracle_kw(cfg):
    return dict(page_size=cfg.page_size, q_pos0=cfg.q_pos0, scale=cfg.scale)


def oracle_bkw(cfg):
    return dict(page_size=cfg.page_size, prefix_len=cfg.prefix_len, q_pos0=cfg.q_pos0,
                scale=cfg.scale)
