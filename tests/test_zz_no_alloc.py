"""The allocation-free sparse forward (ls_sparse_attn_fwd_noalloc) against the
workspace entry point it varies (ls_sparse_attn_fwd): the same kernels, so the
outputs must agree bit for bit, on two calls in a row where the second is
smaller than the first (the scratch array keeps the first call's contents)."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2607_14952_amd import binding as B
from paper_2607_14952_amd import configs, inputs
from paper_2607_14952_amd.replay import to_device
from tests._gpu import announce

pytestmark = pytest.mark.gpu


def _case(cfg, pads=False):
    h = inputs.sparse_inputs(cfg)
    if pads:
        idx = h["idx"].copy()
        idx[1, 5:] = -1
        idx[3, ::2] = -1
        h = dict(h, idx=idx)
    lat = to_device(h["latent_pool"])
    return (to_device(h["q"]), B.PagedKV(lat, lat, to_device(h["page_table"])),
            to_device(h["idx"]) if h["idx"].shape[1] else None)


def test_noalloc_matches_workspace_entry_twice_second_smaller():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()
    big = configs.C5.scaled(name="c5_noalloc_big", prefix_len=65536, resp_len=300, topk=1000)
    small = configs.C5.scaled(name="c5_noalloc_small", prefix_len=8192, resp_len=37, topk=100)
    for cfg, pads in ((big, False), (small, True)):
        q, kv, idx = _case(cfg, pads)
        kw = dict(prefix_len=cfg.prefix_len, q_pos0=cfg.q_pos0, scale=cfg.scale)
        R, H = q.shape[0], q.shape[1]
        announce(f"noalloc {cfg.name}: workspace entry")
        out_a, lse_a = B.sparse_attn_fwd(q, kv, idx, **kw)
        out_b = torch.full((R, H, 512), float("nan"), dtype=torch.float32, device="cuda")
        lse_b = torch.full((H, R), float("nan"), dtype=torch.float32, device="cuda")
        announce(f"noalloc {cfg.name}: allocation-free entry")
        B.sparse_attn_fwd_noalloc(q, kv, idx, out=out_b, lse=lse_b, **kw)
        torch.cuda.synchronize()
        assert torch.equal(out_a, out_b), f"{cfg.name}: out differs"
        assert torch.equal(lse_a, lse_b), f"{cfg.name}: lse differs"


def test_noalloc_rejects_oversize_and_checked_mode_before_launch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cfg = configs.C5.scaled(name="c5_noalloc_reject", prefix_len=8192, resp_len=16, topk=64)
    q, kv, idx = _case(cfg)
    out = torch.empty((16, 128, 512), dtype=torch.float32, device="cuda")
    lse = torch.empty((128, 16), dtype=torch.float32, device="cuda")
    kw = dict(prefix_len=cfg.prefix_len, q_pos0=cfg.q_pos0, scale=cfg.scale)
    with pytest.raises(B.LongStrawError) as ei:
        B.sparse_attn_fwd_noalloc(q, kv, idx, out=out, lse=lse, flags=B.FLAG_CHECKED, **kw)
    assert ei.value.name == "LS_ERR_UNSUPPORTED"
    # 16 rows whose response window is long enough to need more than the scratch:
    # n_q * (topk + window) * 4 bytes > 64 MiB
    big_q0 = cfg.prefix_len + (64 << 20) // (16 * 4)
    n_pages = -(-(big_q0 + 16) // cfg.page_size)
    table = torch.zeros(n_pages, dtype=torch.int32, device="cuda")
    kv_big = B.PagedKV(kv.k_pool, kv.v_pool, table)
    with pytest.raises(B.LongStrawError) as ei:
        B.sparse_attn_fwd_noalloc(q, kv_big, idx, out=out, lse=lse, prefix_len=cfg.prefix_len,
                                  q_pos0=big_q0, scale=cfg.scale)
    assert ei.value.name == "LS_ERR_WORKSPACE"
    torch.cuda.synchronize()
