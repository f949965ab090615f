"""No-grad chunked capture of a prompt into the paged store (one attention layer).

Phase 1 of the replay transaction runs the prompt once with autograd off and
keeps each layer's state; for full attention that state is the K/V pages.  The
prompt is captured in fixed chunks: chunk c = positions [b, e) is written into
its own pages of the pool (ls_scatter_kv through the page table: right-sized
pages that belong to the store, not views of a chunk tensor), then its queries
attend to every earlier position and causally within the chunk
(ls_prefix_attn_fwd over the chunk's splits with q_pos0 = b, then
ls_lse_merge).  Chunking does not change the result: row t's output is causal
attention over positions 0 .. t.
"""
from __future__ import annotations

from . import binding as B


class PrefixCapture:
    """Pools, page table and per-chunk buffers for one capture."""

    def __init__(self, cfg, dev: dict, *, stream=None):
        import torch
        self.cfg = cfg
        self.dev = dev
        self.stream = stream
        S, Hkv, D, Hq = cfg.page_size, cfg.n_kv_heads, cfg.head_dim, cfg.n_q_heads
        bf16 = torch.bfloat16
        dv = dev["k"].device
        # pages start zeroed: pages the table never names stay zero
        self.k_pool = torch.zeros((cfg.n_phys_pages, S, Hkv, D), dtype=bf16, device=dv)
        self.v_pool = torch.zeros((cfg.n_phys_pages, S, Hkv, D), dtype=bf16, device=dv)
        self.kv = B.PagedKV(self.k_pool, self.v_pool, dev["page_table"])
        n_split = max(len(cfg.chunk_splits(c)) for c in range(cfg.n_chunks))
        kw = dict(dtype=torch.float32, device=dv)
        # flat storage, viewed per chunk as contiguous [splits, rows, ...] (a
        # short last chunk needs dense views, not slices of full-chunk ones)
        self._out_part = torch.empty(n_split * cfg.chunk * Hq * D, **kw)
        self._lse_part = torch.empty(n_split * Hq * cfg.chunk, **kw)
        self._lse = torch.empty(Hq * cfg.chunk, **kw)
        self._out = torch.empty(cfg.chunk * Hq * D, dtype=bf16, device=dv)

    def chunk(self, c: int, out=None):
        """Capture chunk c; its attention output goes to ``out`` (rows of the
        chunk, bf16) or to the shared chunk buffer."""
        cfg = self.cfg
        b, e = cfg.chunk_range(c)
        n = e - b
        B.scatter_kv(self.kv, b, self.dev["k"][b:e], self.dev["v"][b:e], stream=self.stream)
        q = self.dev["q_blocks"][c % cfg.n_q_blocks][:n]
        splits = cfg.chunk_splits(c)
        ns = len(splits)
        Hq, D = cfg.n_q_heads, cfg.head_dim
        out_part = self._out_part[:ns * n * Hq * D].view(ns, n, Hq, D)
        lse_part = self._lse_part[:ns * Hq * n].view(ns, Hq, n)
        B.prefix_attn_fwd(q, self.kv, splits, prefix_len=b, q_pos0=b, scale=cfg.scale,
                          out_part=out_part, lse_part=lse_part, stream=self.stream)
        dst = self._out[:n * Hq * D].view(n, Hq, D) if out is None else out
        self.lse = self._lse[:Hq * n].view(Hq, n)
        B.lse_merge(out_part, lse_part, out=dst, lse=self.lse, stream=self.stream)
        return dst

    def run(self):
        for c in range(self.cfg.n_chunks):
            self.chunk(c)
