"""DSA selection for the sparse latent replay: index scores over the prefix and
the top-k of each response row (Eq. dsa-index, Eq. dsa-attention), composed
from ls_dsa_index_scores and ls_topk_select.

``global``: one top-k over each row's scores for the whole prefix.
``candidates``: the prefix is cut into contiguous shards; each shard's local
top-k (with global positions) is a candidate list, and one more top-k over the
concatenated candidates picks the global selection (Eq. glm-global-dsa), the
single-GPU form of the cross-rank candidate merge.  Both give the same indices
(ties go to the lower position in every step).
"""
from __future__ import annotations

from . import binding as B


class DsaSelect:
    def __init__(self, cfg, dev: dict, *, mode: str = "global", n_shards: int = 8, stream=None):
        import torch
        self.cfg = cfg
        self.dev = dev
        self.mode = mode
        self.stream = stream
        R, P, k = cfg.resp_len, cfg.prefix_len, cfg.topk
        ld = P + (-P) % 4
        self.scores = torch.empty((R, ld), dtype=torch.float32, device=dev["q_index"].device)
        self.idx = torch.empty((R, k), dtype=torch.int32, device=self.scores.device)
        self.sel_scores = torch.empty((R, k), dtype=torch.float32, device=self.scores.device)
        if mode == "candidates":
            step = -(-P // n_shards)
            self.shards = [(b, min(P, b + step)) for b in range(0, P, step)]
            self.cand_pos = torch.empty((R, k * len(self.shards)), dtype=torch.int32,
                                        device=self.scores.device)
            self.cand_sc = torch.empty_like(self.cand_pos, dtype=torch.float32)

    def score(self):
        d = self.dev
        B.dsa_index_scores(d["q_index"], d["w_index"], d["k_index_pool"], d["page_table"],
                           pos_begin=0, pos_end=self.cfg.prefix_len, scores=self.scores,
                           stream=self.stream)

    def select(self):
        P, k = self.cfg.prefix_len, self.cfg.topk
        if self.mode == "global":
            B.topk_select(self.scores, k, n=P, out_pos=self.idx, out_scores=self.sel_scores,
                          stream=self.stream)
            return self.idx
        # per-shard candidates (positions ascending across shards), then the merge
        for s, (b, e) in enumerate(self.shards):
            if e - b < k:
                raise ValueError(f"candidate selection: shard [{b}, {e}) holds fewer than "
                                 f"k = {k} positions")
            B.topk_select(self.scores[:, b:], k, n=e - b, pos_offset=b,
                          out_pos=self.cand_pos[:, s * k:(s + 1) * k],
                          out_scores=self.cand_sc[:, s * k:(s + 1) * k], stream=self.stream)
        B.topk_select(self.cand_sc, k, positions=self.cand_pos, out_pos=self.idx,
                      out_scores=self.sel_scores, stream=self.stream)
        return self.idx

    def run(self):
        self.score()
        return self.select()
