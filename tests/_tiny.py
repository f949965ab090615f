"""Tiny hand-built replay problems for oracle pins (float64 unless asked)."""
from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass
class Tiny:
    q: np.ndarray           # [R, Hq, D]
    k_pool: np.ndarray      # [n_phys, S, Hkv, D]
    v_pool: np.ndarray      # [n_phys, S, Hkv, Dv]
    page_table: np.ndarray  # [n_logical] int32
    d_out: np.ndarray       # [R, Hq, Dv]
    S: int
    P: int                  # prefix_len = q_pos0
    scale: float

    @property
    def R(self):
        return self.q.shape[0]

    @property
    def kv_len(self):
        return self.P + self.R

    def kw(self):
        return dict(page_size=self.S, q_pos0=self.P, scale=self.scale)

    def bkw(self):
        return dict(page_size=self.S, prefix_len=self.P, q_pos0=self.P, scale=self.scale)

    def set_rows(self, pool_name, positions, g, values):
        """Write ``values`` into the logical rows ``positions`` of KV head ``g``."""
        pool = getattr(self, pool_name)
        positions = np.asarray(positions)
        pages = self.page_table[positions // self.S]
        pool[pages, positions % self.S, g] = values


def make(P=96, R=12, Hq=4, Hkv=2, D=8, Dv=None, S=16, seed=0, table="perm", extra_pages=3,
         dtype=np.float64, scale=None):
    Dv = D if Dv is None else Dv
    rng = np.random.default_rng(seed)
    n_logical = -(-(P + R) // S)
    n_phys = n_logical + extra_pages
    if table == "identity":
        pt = np.arange(n_logical)
    else:
        pt = rng.permutation(n_phys)[:n_logical]
    return Tiny(
        q=rng.standard_normal((R, Hq, D)).astype(dtype),
        k_pool=rng.standard_normal((n_phys, S, Hkv, D)).astype(dtype),
        v_pool=rng.standard_normal((n_phys, S, Hkv, Dv)).astype(dtype),
        page_table=pt.astype(np.int32),
        d_out=rng.standard_normal((R, Hq, Dv)).astype(dtype),
        S=S, P=P, scale=(1.0 / np.sqrt(D)) if scale is None else scale)


def rel_l2(x, ref):
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(x - ref) / (den if den > 0 else 1.0))
