"""Blockwise response replay against a resident, shared prefix.

The prefix pages stay in one pool for every group member (Sec. "Four-Block
Response Replay"; the resident-prefix runs of Sec. "Lazy Gradient Pages and the
Fixed Eight-H20 Envelope").  A member's response is appended to free pages,
its blocks are replayed in reverse order -- each block's rows attend to the
whole prefix and causally to the response so far -- the response dK/dV
accumulate across blocks (a later block's rows also reach the keys of earlier
blocks), and the pages are popped afterwards.  The prefix pages are never
written and never get a gradient.

Every step runs in the library: ls_scatter_kv (append), ls_prefix_attn_fwd,
ls_lse_merge and ls_prefix_attn_bwd.
"""
from __future__ import annotations

import numpy as np

from . import binding as B
from .replay import to_device


class ResidentPrefix:
    """A paged pool holding a prefix plus free pages for one response at a time."""

    def __init__(self, cfg, store: dict, device="cuda"):
        import torch
        self.cfg = cfg
        self.k_pool = to_device(store["k_pool"], device)
        self.v_pool = to_device(store["v_pool"], device)
        self.table_host = np.zeros(cfg.n_logical_pages, dtype=np.int32)
        self.table_host[:cfg.n_prefix_pages] = store["prefix_table"]
        self.free = list(store["free_pages"].tolist())
        self.table = torch.from_numpy(self.table_host.copy()).to(device)
        self.kv = B.PagedKV(self.k_pool, self.v_pool, self.table)
        self.appended = None

    def append(self, k_resp, v_resp, stream=None):
        """Take response pages from the free list, extend the page table and write
        the response K/V rows at logical positions [prefix_len, prefix_len + R)."""
        import torch
        cfg = self.cfg
        if self.appended is not None:
            raise RuntimeError("a response is already appended; pop it first")
        n = -(-k_resp.shape[0] // cfg.page_size)
        if n > len(self.free):
            raise RuntimeError("pool has no room for the response")
        pages, self.free = self.free[:n], self.free[n:]
        lo = cfg.n_prefix_pages
        self.table_host[lo:lo + n] = pages
        self.table[lo:lo + n].copy_(torch.from_numpy(np.asarray(pages, dtype=np.int32)))
        B.scatter_kv(self.kv, cfg.prefix_len, k_resp, v_resp, stream=stream)
        self.appended = pages

    def pop(self):
        """Return the response pages to the free list (the prefix is untouched)."""
        if self.appended is None:
            raise RuntimeError("nothing appended")
        self.free = list(self.appended) + self.free
        self.appended = None


class BlockwiseReplay:
    """Reverse blockwise replay of one member; buffers are reused across members."""

    def __init__(self, cfg, prefix: ResidentPrefix, stream=None):
        import torch
        self.cfg, self.prefix, self.stream = cfg, prefix, stream
        blk, R = cfg.rows_per_call, cfg.resp_len
        Hq, Hkv, D, Dv = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.head_dim_v
        dev = prefix.k_pool.device
        kw = dict(dtype=torch.float32, device=dev)
        shard = cfg.prefix_len // cfg.n_shards
        self.prefix_ranges = [(s * shard, cfg.prefix_len if s == cfg.n_shards - 1 else (s + 1) * shard)
                              for s in range(cfg.n_shards)]
        # the forward's prefix splits: each shard range cut splits_per_shard ways, so
        # a launch holds many equal workgroups; the backward runs once per shard range
        self.fwd_ranges = cfg.splits()[:-1]
        n_parts = len(self.fwd_ranges) + 1
        self.n_parts = n_parts
        self.out_part_flat = torch.empty(n_parts * blk * Hq * Dv, **kw)
        self.lse_part_flat = torch.empty(n_parts * Hq * blk, **kw)
        self.out_flat = torch.empty(blk * Hq * Dv, dtype=prefix.k_pool.dtype, device=dev)
        self.lse_flat = torch.empty(Hq * blk, **kw)
        self.dq = torch.empty((R, Hq, D), **kw)
        self.dk = torch.zeros((R, Hkv, D), **kw)
        self.dv = torch.zeros((R, Hkv, Dv), **kw)
        self.ws = None

    def block_rows(self, b):
        blk = self.cfg.rows_per_call
        return slice(b * blk, min((b + 1) * blk, self.cfg.resp_len))

    def run_block(self, b, q, d_out, keep=None, first=False):
        """Forward, merge and backward of block b (rows block_rows(b)).  The first
        block replayed (the last one) writes the response dK/dV, later ones add."""
        c = self.cfg
        rows = self.block_rows(b)
        qb, dob = q[rows], d_out[rows]
        q0 = c.prefix_len + rows.start
        kv_end = q0 + qb.shape[0]
        splits = self.fwd_ranges + [(c.prefix_len, kv_end)]
        n = qb.shape[0]
        Hq, Dv, P = c.n_q_heads, c.head_dim_v, self.n_parts
        op = self.out_part_flat[:P * n * Hq * Dv].view(P, n, Hq, Dv)
        lp = self.lse_part_flat[:P * Hq * n].view(P, Hq, n)
        B.prefix_attn_fwd(qb, self.prefix.kv, splits, prefix_len=c.prefix_len, q_pos0=q0,
                          scale=c.scale, out_part=op, lse_part=lp, stream=self.stream)
        out = self.out_flat[:n * Hq * Dv].view(n, Hq, Dv)
        lse = self.lse_flat[:Hq * n].view(Hq, n)
        B.lse_merge(op, lp, out=out, lse=lse, stream=self.stream)
        if keep is not None:
            keep[b] = (out.clone(), lse.clone())
        if self.ws is None:   # sized for the block with the most response keys (highest q_pos0)
            self.ws = B.bwd_workspace(q[:c.rows_per_call], self.prefix.kv, prefix_len=c.prefix_len,
                                      q_pos0=c.prefix_len + (c.blocks - 1) * c.rows_per_call)
        dq = self.dq[rows]
        for r, (kb, ke) in enumerate(self.prefix_ranges + [(c.prefix_len, kv_end)]):
            B.prefix_attn_bwd(qb, self.prefix.kv, dob, out, lse, prefix_len=c.prefix_len,
                              q_pos0=q0, scale=c.scale, kv_begin=kb, kv_end=ke,
                              flags=((B.FLAG_ACCUMULATE_DQ | B.FLAG_PREP_READY) if r else 0)
                              | (0 if first else B.FLAG_ACCUMULATE_DKV),
                              dq=dq, dk_resp=self.dk[:kv_end - c.prefix_len],
                              dv_resp=self.dv[:kv_end - c.prefix_len], workspace=self.ws,
                              stream=self.stream)

    def run_member(self, resp_dev: dict, keep=None, block_events=None):
        """append -> blocks in reverse -> pop; returns (dq, dk, dv) of the member.
        block_events: optional {b: (start, end)} timing events, recorded on the
        replay's stream around each block."""
        self.prefix.append(resp_dev["k"], resp_dev["v"], stream=self.stream)
        last = self.cfg.blocks - 1
        for b in reversed(range(self.cfg.blocks)):
            if block_events is not None:
                block_events[b][0].record(self.stream)
            self.run_block(b, resp_dev["q"], resp_dev["d_out"], keep=keep, first=(b == last))
            if block_events is not None:
                block_events[b][1].record(self.stream)
        self.prefix.pop()
        return self.dq, self.dk, self.dv


def block_flops(cfg, b):
    """FLOP convention of the replay step for block b (rows attend to the prefix
    and causally to the response up to themselves)."""
    blk = cfg.rows_per_call
    r0 = b * blk
    n = min(blk, cfg.resp_len - r0)
    pre = n * cfg.prefix_len
    resp = sum(r0 + i + 1 for i in range(n))
    Hq, D = cfg.n_q_heads, cfg.head_dim
    return 4 * Hq * D * (pre + resp), Hq * D * (6 * pre + 10 * resp)
