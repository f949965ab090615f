"""Workload registry for response-replay attention.

Each entry describes the shape of one replay problem: a response suffix of
``resp_len`` query tokens, causal among themselves, attending to a paged KV
prefix of ``prefix_len`` positions (stop-gradient state, Sec. "Conditional
Replay as an Efficiency Boundary", Eq. gradient-boundary).  The prefix is cut
into ``n_shards`` contiguous KV ranges (the single-GPU stand-in for the
context-parallel ranks of Sec. "Global Full-Attention Forward Composition"),
each of which is further split ``splits_per_shard`` ways; the response keys
form one extra split.

Nothing here computes attention: these are shapes, seeds and input recipes.
"""
from __future__ import annotations

import dataclasses
import math


@dataclasses.dataclass(frozen=True)
class ReplayConfig:
    name: str
    seed: int
    dtype: str                 # "bf16" or "f32": q, K/V pools and dO
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    head_dim_v: int
    page_size: int
    prefix_len: int
    resp_len: int              # response tokens (causal among themselves)
    n_shards: int = 1
    splits_per_shard: int = 1
    table: str = "perm"        # "identity" | "perm" | "sample"
    pool_slack: float = 1.0    # physical pages / logical pages (>= 1)
    plant_frac: float = 0.0    # fraction of prefix keys aligned to a random query
    plant_gain: float = 4.0
    backward: bool = True
    sparse: bool = False       # MLA/DSA latent replay (one shared latent row)
    topk: int = 0
    members: int = 1           # responses replayed against one prefix pool
    block: int = 0             # rows per replay call in blockwise replay (0 = whole response)

    # -- derived sizes ---------------------------------------------------
    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def q_pos0(self) -> int:
        return self.prefix_len

    @property
    def kv_len(self) -> int:
        return self.prefix_len + self.resp_len

    @property
    def rows_per_call(self) -> int:
        return self.block or self.resp_len

    @property
    def blocks(self) -> int:
        return -(-self.resp_len // self.rows_per_call)

    @property
    def n_prefix_pages(self) -> int:
        return -(-self.prefix_len // self.page_size)

    @property
    def n_resp_pages(self) -> int:
        return -(-self.resp_len // self.page_size)

    @property
    def n_logical_pages(self) -> int:
        return self.n_prefix_pages + self.n_resp_pages

    @property
    def n_phys_pages(self) -> int:
        # Members replay one at a time, so one response's pages are live at once;
        # a pool with slack takes them from its free pages.
        return max(math.ceil(self.n_prefix_pages * self.pool_slack - 1e-9),
                   self.n_prefix_pages + self.n_resp_pages)

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    def splits(self):
        """Logical key ranges [begin, end): n_shards x splits_per_shard over the
        prefix, then one split holding the response keys."""
        out = []
        shard = self.prefix_len // self.n_shards
        for s in range(self.n_shards):
            b0 = s * shard
            e0 = self.prefix_len if s == self.n_shards - 1 else b0 + shard
            step = -(-(e0 - b0) // self.splits_per_shard)
            b = b0
            while b < e0:
                e = min(e0, b + step)
                out.append((b, e))
                b = e
        out.append((self.prefix_len, self.kv_len))
        return out

    def shard_ranges(self):
        shard = self.prefix_len // self.n_shards
        out = [(s * shard, self.prefix_len if s == self.n_shards - 1 else (s + 1) * shard)
               for s in range(self.n_shards)]
        out.append((self.prefix_len, self.kv_len))
        return out

    def scaled(self, **kw) -> "ReplayConfig":
        return dataclasses.replace(self, **kw)


# Tiny fp32 replay: correctness only.
C1 = ReplayConfig(name="c1_tiny_f32", seed=1, dtype="f32", n_q_heads=2, n_kv_heads=1,
                  head_dim=64, head_dim_v=64, page_size=64, prefix_len=4096, resp_len=128,
                  n_shards=2, splits_per_shard=1, table="identity")

# Forward-only single shard: one eighth of a 2M prefix.
C2 = ReplayConfig(name="c2_fwd_262k", seed=2, dtype="bf16", n_q_heads=16, n_kv_heads=2,
                  head_dim=256, head_dim_v=256, page_size=256, prefix_len=262_144,
                  resp_len=4096, n_shards=1, splits_per_shard=1, table="perm", backward=False)

# Full 2M replay, 8 contiguous shards x 4-way split-KV + the response split.
C3 = ReplayConfig(name="c3_replay_2m", seed=3, dtype="bf16", n_q_heads=16, n_kv_heads=2,
                  head_dim=256, head_dim_v=256, page_size=256, prefix_len=2_097_152,
                  resp_len=4096, n_shards=8, splits_per_shard=4, table="perm",
                  plant_frac=0.01)

# 4.46M resident prefix, 8 members of 8,192 tokens replayed in 2,048-token blocks.
C4 = ReplayConfig(name="c4_resident_4p46m_g8", seed=4, dtype="bf16", n_q_heads=16,
                  n_kv_heads=2, head_dim=256, head_dim_v=256, page_size=256,
                  prefix_len=4_456_448, resp_len=8192, n_shards=8, splits_per_shard=1,
                  table="sample", pool_slack=1.125, members=8, block=2048)

# MLA/DSA-style sparse latent replay.
C5 = ReplayConfig(name="c5_sparse_mla_2m", seed=5, dtype="bf16", n_q_heads=128, n_kv_heads=1,
                  head_dim=576, head_dim_v=512, page_size=64, prefix_len=2_097_152,
                  resp_len=2048, table="perm", sparse=True, topk=2048)

CONFIGS = {c.name: c for c in (C1, C2, C3, C4, C5)}
BY_SHORT = {"c1": C1, "c2": C2, "c3": C3, "c4": C4, "c5": C5}


def get(name: str) -> ReplayConfig:
    return BY_SHORT.get(name) or CONFIGS[name]
