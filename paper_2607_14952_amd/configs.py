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
    plant_unit: bool = False   # add gain * q / |q| instead of gain * q (the literal "+4 sigma" reading)
    backward: bool = True
    sparse: bool = False       # MLA/DSA latent replay (one shared latent row)
    topk: int = 0
    members: int = 1           # responses replayed against one prefix pool
    block: int = 0             # rows per replay call in blockwise replay (0 = whole response)
    index_heads: int = 0           # sparse: DSA index heads (Eq. dsa-index, width 128) selecting
                                   # the top-k; 0 = seeded indices
    ownership: str = "contiguous"  # "contiguous" ranges or "cyclic": page p to shard p mod n_shards
    bf16_numerator: bool = False   # cross-shard merge reduces the numerator in bf16

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

    def shard_pages(self, shard: int):
        """Logical prefix pages of ``shard`` under cyclic ownership (Eq.
        qwen-page-owner: owner(p) = p mod n_shards), in increasing order."""
        return list(range(shard, self.n_prefix_pages, self.n_shards))

    def shard_len(self, shard: int) -> int:
        """Prefix positions owned by ``shard`` under cyclic ownership."""
        pages = self.shard_pages(shard)
        if not pages:
            return 0
        last = min(self.page_size, self.prefix_len - pages[-1] * self.page_size)
        return (len(pages) - 1) * self.page_size + last

    def virtual_splits(self, shard: int):
        """Cyclic ownership: the shard's ``splits_per_shard`` ranges over its
        owned positions renumbered 0 .. shard_len - 1 (page i of the shard's
        table is its i-th owned page)."""
        n = self.shard_len(shard)
        step = -(-n // self.splits_per_shard) if n else 1
        return [(b, min(n, b + step)) for b in range(0, n, step)]

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

# Forward-only single shard: one eighth of a 2M prefix, cut into 4 splits like
# each shard of c3 (a single split leaves half the workgroups short).
C2 = ReplayConfig(name="c2_fwd_262k", seed=2, dtype="bf16", n_q_heads=16, n_kv_heads=2,
                  head_dim=256, head_dim_v=256, page_size=256, prefix_len=262_144,
                  resp_len=4096, n_shards=1, splits_per_shard=4, table="perm", backward=False)

# Full 2M replay, 8 contiguous shards x 4-way split-KV + the response split.
C3 = ReplayConfig(name="c3_replay_2m", seed=3, dtype="bf16", n_q_heads=16, n_kv_heads=2,
                  head_dim=256, head_dim_v=256, page_size=256, prefix_len=2_097_152,
                  resp_len=4096, n_shards=8, splits_per_shard=4, table="perm",
                  plant_frac=0.01)

# 4.46M resident prefix, 8 members of 8,192 tokens replayed in 2,048-token blocks.
C4 = ReplayConfig(name="c4_resident_4p46m_g8", seed=4, dtype="bf16", n_q_heads=16,
                  n_kv_heads=2, head_dim=256, head_dim_v=256, page_size=256,
                  prefix_len=4_456_448, resp_len=8192, n_shards=8, splits_per_shard=8,
                  table="sample", pool_slack=1.125, members=8, block=2048)

# MLA/DSA-style sparse latent replay.
C5 = ReplayConfig(name="c5_sparse_mla_2m", seed=5, dtype="bf16", n_q_heads=128, n_kv_heads=1,
                  head_dim=576, head_dim_v=512, page_size=64, prefix_len=2_097_152,
                  resp_len=2048, table="perm", sparse=True, topk=2048)



@dataclasses.dataclass(frozen=True)
class CaptureConfig:
    """No-grad chunked capture of a prompt into a paged store, one attention
    layer (Phase 1 of the replay transaction; the shared prompt is captured in
    4,096-token chunks, Sec. "Four-Block Response Replay").  Chunk c's queries
    attend to every earlier position and causally within the chunk; its K/V
    rows are copied into pages of their own (right-sized pages, Sec. "From
    Logical Shards to Physical Pages")."""
    name: str
    seed: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    page_size: int
    length: int                    # prompt positions captured
    chunk: int                     # positions per capture chunk
    # earlier-chunk keys per split of a chunk's forward: short splits give every chunk
    # many equal workgroups (the last chunk 64 pieces + its own), which keeps all CUs busy
    keys_per_split: int = 32_768
    q_blocks: int = 0              # distinct query blocks; chunk c uses block c mod q_blocks (0: own)
    pool_slack: float = 1.0
    table: str = "perm"
    dtype: str = "bf16"

    @property
    def head_dim_v(self) -> int:
        return self.head_dim

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def n_chunks(self) -> int:
        return -(-self.length // self.chunk)

    @property
    def n_logical_pages(self) -> int:
        return -(-self.length // self.page_size)

    @property
    def n_phys_pages(self) -> int:
        return max(self.n_logical_pages, math.ceil(self.n_logical_pages * self.pool_slack - 1e-9))

    @property
    def n_q_blocks(self) -> int:
        return self.q_blocks or self.n_chunks

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    def chunk_range(self, c: int):
        return c * self.chunk, min(self.length, (c + 1) * self.chunk)

    def chunk_splits(self, c: int):
        """Key ranges of chunk c's forward: the earlier positions in pieces of
        at most keys_per_split, then the chunk's own positions (causal)."""
        b, e = self.chunk_range(c)
        n = -(-b // self.keys_per_split) if b else 0
        step = -(-b // n) if n else 0
        out = [(s, min(b, s + step)) for s in range(0, b, step)] if n else []
        out.append((b, e))
        return out

    def visible(self) -> int:
        """Sum over captured rows of the keys each sees (positions 0 .. t)."""
        return self.length * (self.length + 1) // 2


# One attention layer's capture of a 2,097,152-position prompt in 512 chunks of
# 4,096 (the c3 layer shape); eight query blocks are cycled (query values do
# not change the work).
CAPTURE_2M = CaptureConfig(name="capture_2m", seed=6, n_q_heads=16, n_kv_heads=2, head_dim=256,
                           page_size=256, length=2_097_152, chunk=4096, q_blocks=8)

CONFIGS = {c.name: c for c in (C1, C2, C3, C4, C5)}
BY_SHORT = {"c1": C1, "c2": C2, "c3": C3, "c4": C4, "c5": C5}


def get(name: str):
    if name in ("capture", CAPTURE_2M.name):
        return CAPTURE_2M
    return BY_SHORT.get(name) or CONFIGS[name]
