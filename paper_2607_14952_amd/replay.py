"""One response-replay step over a paged prefix, composed from the library calls.

forward  : every split's local (o_r, l_r)        -> ls_prefix_attn_fwd (one launch)
           splits of a shard -> shard (o_s, l_s)  -> ls_lse_merge (fp32)
           shards + response -> global (o, l)     -> ls_lse_merge (q dtype; with
           bf16_numerator the numerator is reduced in bf16, as the production
           composition noted after Eq. qwen-global-attn)
           (the single-GPU form of the cross-rank merge, Eq. qwen-lse-parts and
           Eq. qwen-global-attn)
backward : per shard key range, dq accumulated in shard order (Eq. qwen-dq-reduce);
           the response range also yields the response dK/dV (lazy gradient pages:
           prefix keys get none).

Shards own contiguous prefix ranges, or, with ``ownership="cyclic"``, the pages
p with p mod n_shards = c (Eq. qwen-page-owner).  A cyclic shard gets a page
table of its own whose first entries are its owned pages in order, so its keys
form one range 0 .. shard_len - 1 of that table, and it takes one forward launch
and one backward call.  Renumbering is exact here because every prefix position
precedes every query row, so each prefix key is visible to each row whatever
its position; the response split keeps the global table and coordinates.
"""
from __future__ import annotations

import numpy as np

from . import binding as B


def to_device(arr: np.ndarray, device="cuda"):
    """numpy input (uint16 bf16 bit patterns, float32 or int32) -> torch device tensor."""
    import torch
    if arr.dtype == np.uint16:
        return torch.from_numpy(arr.view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(arr)).to(device)


def device_inputs(host: dict, device="cuda") -> dict:
    out = {}
    for k in ("q", "k_pool", "v_pool", "page_table", "d_out", "latent_pool", "idx"):
        if k in host:
            out[k] = to_device(host[k], device)
    return out


class ReplayStep:
    """Buffers and call sequence of one fwd(+bwd) replay over a config's shards."""

    def __init__(self, cfg, dev: dict, *, backward: bool | None = None, stream=None):
        import torch
        self.cfg = cfg
        self.dev = dev
        self.kv = B.PagedKV(dev["k_pool"], dev["v_pool"], dev["page_table"])
        self.backward_enabled = cfg.backward if backward is None else backward
        self.stream = stream
        q = dev["q"]
        R, Hq, D, Dv = cfg.resp_len, cfg.n_q_heads, cfg.head_dim, cfg.head_dim_v
        self.cyclic = cfg.ownership == "cyclic"
        if self.cyclic:
            # per shard: its own PagedKV (owned pages first) and its virtual ranges;
            # the response shard keeps the global table
            table = dev["page_table"].cpu().numpy()
            self.shard_kv, self.shard_splits, self.shards = [], [], []
            for c in range(cfg.n_shards):
                n = cfg.shard_len(c)
                if n == 0:
                    continue
                t = table.copy()
                pages = cfg.shard_pages(c)
                t[:len(pages)] = table[pages]
                self.shard_kv.append(B.PagedKV(dev["k_pool"], dev["v_pool"],
                                               torch.from_numpy(t).to(q.device)))
                self.shard_splits.append(cfg.virtual_splits(c))
                self.shards.append((0, n))
            self.shard_kv.append(self.kv)
            self.shard_splits.append([(cfg.prefix_len, cfg.kv_len)])
            self.shards.append((cfg.prefix_len, cfg.kv_len))
            self.splits = [r for sp in self.shard_splits for r in sp]
        else:
            self.splits = [r for r in cfg.splits() if r[0] < r[1]]
            self.shards = [r for r in cfg.shard_ranges() if r[0] < r[1]]
        kw = dict(dtype=torch.float32, device=q.device)
        self.out_part = torch.empty((len(self.splits), R, Hq, Dv), **kw)
        self.lse_part = torch.empty((len(self.splits), Hq, R), **kw)
        self.shard_out = torch.empty((len(self.shards), R, Hq, Dv), **kw)
        self.shard_lse = torch.empty((len(self.shards), Hq, R), **kw)
        self.out = torch.empty((R, Hq, Dv), dtype=q.dtype, device=q.device)
        self.lse = torch.empty((Hq, R), **kw)
        # which splits belong to which shard (splits are listed shard by shard)
        self.groups = []
        i = 0
        if self.cyclic:
            for sp in self.shard_splits:
                self.groups.append((i, i + len(sp)))
                i += len(sp)
        else:
            for b, e in self.shards:
                j = i
                while j < len(self.splits) and self.splits[j][1] <= e:
                    j += 1
                self.groups.append((i, j))
                i = j
        assert i == len(self.splits)
        if self.backward_enabled:
            self.dq = torch.empty((R, Hq, D), **kw)
            self.dk = torch.zeros((cfg.kv_len - cfg.prefix_len, cfg.n_kv_heads, D), **kw)
            self.dv = torch.zeros((cfg.kv_len - cfg.prefix_len, cfg.n_kv_heads, Dv), **kw)
            self.ws = B.bwd_workspace(q, self.kv, prefix_len=cfg.prefix_len, q_pos0=cfg.q_pos0)

    def forward_splits(self):
        """Local (o_r, l_r) of every split: one launch (one per shard when cyclic)."""
        c = self.cfg
        kw = dict(prefix_len=c.prefix_len, q_pos0=c.q_pos0, scale=c.scale, stream=self.stream)
        if not self.cyclic:
            B.prefix_attn_fwd(self.dev["q"], self.kv, self.splits, out_part=self.out_part,
                              lse_part=self.lse_part, **kw)
            return
        for s, (i, j) in enumerate(self.groups):
            B.prefix_attn_fwd(self.dev["q"], self.shard_kv[s], self.shard_splits[s],
                              out_part=self.out_part[i:j], lse_part=self.lse_part[i:j], **kw)

    def merge(self):
        """Splits -> per-shard results (fp32) -> global result (q dtype)."""
        for s, (i, j) in enumerate(self.groups):
            B.lse_merge(self.out_part[i:j], self.lse_part[i:j], out=self.shard_out[s],
                        lse=self.shard_lse[s], stream=self.stream)
        B.lse_merge(self.shard_out, self.shard_lse, out=self.out, lse=self.lse,
                    flags=B.FLAG_BF16_NUMERATOR if self.cfg.bf16_numerator else 0,
                    stream=self.stream)

    def forward(self):
        self.forward_splits()
        self.merge()
        return self.out, self.lse

    def backward_range(self, r: int):
        """dq contribution of shard range r (accumulated after the first range);
        the response range also writes the response dK/dV.  Ranges after the
        first reuse the Delta and lse * log2(e) the first one left in the
        workspace, so ranges must run in order, starting at 0."""
        c = self.cfg
        b, e = self.shards[r]
        kv = self.shard_kv[r] if self.cyclic else self.kv
        B.prefix_attn_bwd(self.dev["q"], kv, self.dev["d_out"], self.out, self.lse,
                          prefix_len=c.prefix_len, q_pos0=c.q_pos0, scale=c.scale,
                          kv_begin=b, kv_end=e,
                          flags=(B.FLAG_ACCUMULATE_DQ | B.FLAG_PREP_READY) if r > 0 else 0,
                          dq=self.dq, dk_resp=self.dk, dv_resp=self.dv, workspace=self.ws,
                          stream=self.stream)

    def backward(self):
        for r in range(len(self.shards)):
            self.backward_range(r)
        return self.dq, self.dk, self.dv

    def step(self):
        self.forward()
        if self.backward_enabled:
            self.backward()
