"""Page and pool arithmetic of the configurations against the figures the paper
prints for its 2M-context layouts (tests/golden/page_arithmetic.json, cited
there).  CPU only."""
from __future__ import annotations

import json
import os

import numpy as np

from paper_2607_14952_amd import configs, inputs

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "page_arithmetic.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def _page_bytes(page_size, n_kv_heads, head_dim):
    """Bytes of one physical page of a bf16 pool as inputs.py lays it out."""
    tiny = configs.C3.scaled(name="golden_tiny", prefix_len=2 * page_size, resp_len=1,
                             page_size=page_size, n_kv_heads=n_kv_heads, n_q_heads=n_kv_heads,
                             head_dim=head_dim, head_dim_v=head_dim, n_shards=1,
                             splits_per_shard=1, plant_frac=0.0)
    pool = inputs._pool(tiny, 1, head_dim, n_kv_heads)
    return pool.nbytes // tiny.n_phys_pages


def test_qwen_cp8_page_count_and_kv_bytes():
    g = _golden()["qwen_cp8"]
    cfg = configs.C3.scaled(name="golden_qwen", prefix_len=g["prompt_tokens"],
                            resp_len=g["response_tokens"], page_size=g["page_size"],
                            n_kv_heads=g["kv_heads"], n_q_heads=4 * g["kv_heads"],
                            head_dim=g["head_dim"], head_dim_v=g["head_dim"], plant_frac=0.0)
    assert cfg.kv_len == g["context_length"]
    assert cfg.n_prefix_pages == g["prompt_pages"]
    owned = np.bincount(np.arange(cfg.n_prefix_pages) % g["cp_ranks"], minlength=g["cp_ranks"])
    assert (owned == g["pages_per_rank"]).all()
    per_page = _page_bytes(g["page_size"], g["kv_heads"], g["head_dim"])
    assert per_page == g["page_size"] * g["kv_heads"] * g["head_dim"] * g["bytes_per_element"]
    kv_bytes = g["full_attention_layers"] * int(owned[0]) * 2 * per_page   # K and V pools
    assert kv_bytes == g["kv_bytes_per_rank"]


def test_glm_cp32_pages_per_rank():
    g = _golden()["glm_cp32"]
    cfg = configs.C5
    assert cfg.prefix_len == g["prefix_len"] and cfg.page_size == g["page_size"]
    assert cfg.n_prefix_pages // g["cp_ranks"] == g["pages_per_rank"]
    assert cfg.n_prefix_pages % g["cp_ranks"] == 0
    assert g["pages_per_rank"] * cfg.page_size == g["tokens_per_rank"]
