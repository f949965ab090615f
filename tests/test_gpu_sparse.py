"""Sparse latent replay (MLA/DSA): HIP path vs the fp64 oracle (needs an MI355X).

Bars: out rel-L2 <= 5e-3, lse max-abs <= 1e-3, dq rel-L2 <= 1e-2 (bf16 inputs)."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2607_14952_amd import binding as B
from paper_2607_14952_amd import configs, inputs
from paper_2607_14952_amd.replay import to_device
from tests import _par
from tests._gpu import announce, host, lse_err, rel_l2

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu_ready():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()


def run(cfg, h, *, q_pos0=None, rows=None, backward=True, out_bf16=True):
    import torch
    q_pos0 = cfg.prefix_len if q_pos0 is None else q_pos0
    q = to_device(h["q"])
    lat = to_device(h["latent_pool"])
    kv = B.PagedKV(lat, lat, to_device(h["page_table"]))
    idx = to_device(h["idx"]) if h["idx"].shape[1] else None
    announce(f"sparse {cfg.name} R={h['q'].shape[0]} topk={h['idx'].shape[1]} q_pos0={q_pos0}")
    out, lse = B.sparse_attn_fwd(q, kv, idx, prefix_len=cfg.prefix_len, q_pos0=q_pos0,
                                 scale=cfg.scale)
    dq = None
    if backward:
        out_b = out.to(torch.bfloat16) if out_bf16 else out
        dq = B.sparse_attn_bwd(q, kv, idx, to_device(h["d_out"]), out_b, lse,
                               prefix_len=cfg.prefix_len, q_pos0=q_pos0, scale=cfg.scale)
    torch.cuda.synchronize()
    kw = dict(page_size=cfg.page_size, prefix_len=cfg.prefix_len, q_pos0=q_pos0, scale=cfg.scale)
    r = np.arange(h["q"].shape[0]) if rows is None else np.asarray(rows)
    o_ref, l_ref, dq_ref = _par.sparse(h, rows=r, backward=backward, **kw)
    assert rel_l2(host(out)[r], o_ref) <= 5e-3, "sparse out"
    assert lse_err(host(lse)[:, r], l_ref) <= 1e-3, "sparse lse"
    if backward:
        assert rel_l2(host(dq)[r], dq_ref) <= 1e-2, f"sparse dq {rel_l2(host(dq)[r], dq_ref):.2e}"


SMALL = configs.C5.scaled(name="c5_small", prefix_len=8192, resp_len=70, topk=300)


def test_sparse_small():
    run(SMALL, inputs.sparse_inputs(SMALL))


def test_sparse_fp32_output_to_backward():
    """The backward takes the forward's fp32 output as it was written (Delta
    from fp32 O), as the sparse replay benchmark does."""
    run(SMALL.scaled(name="c5_small_o32"), inputs.sparse_inputs(SMALL), out_bf16=False)


def test_sparse_window_only_and_offset_rows():
    """topk = 0 (only the response window), and rows that start after earlier
    response positions (q_pos0 > prefix_len: the window reaches back to prefix_len)."""
    cfg = SMALL.scaled(name="c5_win", topk=0, resp_len=40)
    h = inputs.sparse_inputs(cfg)
    run(cfg, h)
    cfg2 = SMALL.scaled(name="c5_off", resp_len=33, topk=64)
    h2 = inputs.sparse_inputs(cfg2.scaled(resp_len=33 + 50))   # pool holds 50 earlier response rows
    h2 = dict(h2, q=h2["q"][50:], d_out=h2["d_out"][50:], idx=h2["idx"][50:])
    run(cfg2, h2, q_pos0=cfg2.prefix_len + 50)


def test_sparse_two_head_groups():
    """256 query heads: two workgroups per token (grid y = head group), each
    over its own 128 heads of the shared latent rows; a response length that
    is not a multiple of anything the kernels tile by."""
    cfg = SMALL.scaled(name="c5_256h", n_q_heads=256, resp_len=23, topk=97)
    run(cfg, inputs.sparse_inputs(cfg))


def test_sparse_two_to_four_tiles():
    """Key lists of 33 .. 128 entries (2, 3 and 4 tiles of 32): the forward
    keeps three tiles in flight, so these tokens end inside its prologue or its
    first iterations, where later tiles are clamped to the last one."""
    cfg = SMALL.scaled(name="c5_few_tiles", resp_len=96, topk=32)
    run(cfg, inputs.sparse_inputs(cfg))


def test_sparse_invalid_entries_select_nothing():
    """Selections padded with -1 (what the top-k writes for a row with fewer
    candidates than k) and entries at or past the prefix select no key: a row
    of pads only, rows with pads interleaved, rows whose pads fill whole tiles,
    and response positions inside the selection.  The oracle drops the same
    entries."""
    cfg = SMALL.scaled(name="c5_pads", resp_len=40, topk=160)
    h = inputs.sparse_inputs(cfg)
    idx = h["idx"].copy()
    rng = np.random.default_rng(9)
    idx[0] = -1                                    # only the response window
    idx[1, 100:] = -1                              # a short selection, padded at the end
    idx[2, ::3] = -1                               # pads interleaved
    idx[3, :64] = -1                               # two whole tiles of pads first
    idx[4, 10:20] = cfg.prefix_len + np.arange(10) # response positions: no key
    idx[5, 5] = cfg.prefix_len + 39                # a position past this row's window
    idx[6, 7] = -7                                 # another negative value
    idx[7] = np.sort(rng.choice(cfg.prefix_len, cfg.topk, replace=False))
    h = dict(h, idx=idx)
    run(cfg, h)


def test_sparse_checked_mode_index_validation():
    """Checked mode accepts -1 pads and rejects duplicates and other values
    outside the prefix, before launching anything."""
    import torch
    cfg = SMALL.scaled(name="c5_checked", resp_len=8, topk=64)
    h = inputs.sparse_inputs(cfg)
    q = to_device(h["q"])
    lat = to_device(h["latent_pool"])
    kv = B.PagedKV(lat, lat, to_device(h["page_table"]))
    kw = dict(prefix_len=cfg.prefix_len, q_pos0=cfg.q_pos0, scale=cfg.scale, flags=B.FLAG_CHECKED)
    announce("sparse checked mode")
    ok = h["idx"].copy()
    ok[2, 40:] = -1
    B.sparse_attn_fwd(q, kv, to_device(ok), **kw)
    torch.cuda.synchronize()
    for bad, what in ((lambda a: a.__setitem__((3, 5), a[3, 4]), "duplicate"),
                      (lambda a: a.__setitem__((1, 0), -2), "-2"),
                      (lambda a: a.__setitem__((0, 9), cfg.prefix_len), "prefix_len")):
        x = h["idx"].copy()
        bad(x)
        with pytest.raises(B.LongStrawError) as ei:
            B.sparse_attn_fwd(q, kv, to_device(x), **kw)
        assert ei.value.name == "LS_ERR_INVALID_ARG", what


@pytest.mark.timeout(900)
def test_c5_full_size():
    """c5 as bench.py times it: every row's out, lse and dq."""
    cfg = configs.C5
    run(cfg, inputs.sparse_inputs(cfg))
