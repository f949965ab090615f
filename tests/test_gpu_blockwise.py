"""Blockwise replay against a resident prefix (append -> reverse blocks -> pop)
vs the fp64 oracle of the unblocked response (needs an MI355X)."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2607_14952_amd import binding as B
from paper_2607_14952_amd import configs, inputs
from paper_2607_14952_amd.blockwise import BlockwiseReplay, ResidentPrefix
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


def logical_store(cfg, store, resp, pages):
    """Host pools with the response rows written at logical positions
    [prefix_len, prefix_len + R) of the extended table (input layout only)."""
    table = np.concatenate([store["prefix_table"], np.asarray(pages, np.int32)])
    kp, vp = store["k_pool"].copy(), store["v_pool"].copy()
    j = cfg.prefix_len + np.arange(cfg.resp_len)
    kp[table[j // cfg.page_size], j % cfg.page_size] = resp["k"]
    vp[table[j // cfg.page_size], j % cfg.page_size] = resp["v"]
    return kp, vp, table


def run_members(cfg, members, rows=None, keys=None, dq_rows=None, kv_head=None):
    """Replay each member blockwise and compare out/lse on ``rows``, dq on
    ``dq_rows`` (default: ``rows``) and dK/dV on ``keys`` (default: all response
    keys) with the oracle of the unblocked response over the same logical store.
    ``kv_head`` restricts every comparison to that KV head and its group's query
    heads (the oracle then computes only those)."""
    import torch
    store = inputs.prefix_store(cfg)
    prefix = ResidentPrefix(cfg, store)
    rep = BlockwiseReplay(cfg, prefix)
    # device snapshot of the prefix pages and of the table's prefix entries
    pp = torch.from_numpy(store["prefix_table"].astype(np.int64)).to(prefix.k_pool.device)
    k_snap = prefix.k_pool.index_select(0, pp)
    v_snap = prefix.v_pool.index_select(0, pp)
    t_snap = prefix.table[:cfg.n_prefix_pages].clone()
    R = cfg.resp_len
    r_sel = np.arange(R) if rows is None else np.unique(rows)
    dq_sel = r_sel if dq_rows is None else np.unique(np.asarray(dq_rows, np.int64))
    key_off = np.arange(R) if keys is None else np.unique(keys)
    for m in members:
        resp = inputs.response_inputs(cfg, m)
        dev = {k: to_device(v) for k, v in resp.items()}
        pages = prefix.free[:cfg.n_resp_pages]
        keep = {}
        announce(f"{cfg.name} member {m}")
        dq, dk, dv = rep.run_member(dev, keep=keep)
        torch.cuda.synchronize()
        kp, vp, table = logical_store(cfg, store, resp, pages)
        hh = dict(q=resp["q"], k_pool=kp, v_pool=vp, page_table=table, d_out=resp["d_out"])
        kw = dict(page_size=cfg.page_size, q_pos0=cfg.prefix_len, scale=cfg.scale,
                  prefix_len=cfg.prefix_len)
        G = cfg.n_q_heads // cfg.n_kv_heads
        heads = (np.arange(cfg.n_q_heads) if kv_head is None
                 else np.arange(kv_head * G, (kv_head + 1) * G))
        kvh = np.arange(cfg.n_kv_heads) if kv_head is None else np.array([kv_head])
        need = np.union1d(np.union1d(r_sel, dq_sel), np.arange(int(key_off.min()), R))
        o_n, l_n = _par.dense_fwd(hh, rows=need, heads=None if kv_head is None else heads, **kw)
        at = np.searchsorted(need, r_sel)
        out = np.concatenate([host(keep[b][0]) for b in range(cfg.blocks)])
        lse = np.concatenate([host(keep[b][1]) for b in range(cfg.blocks)], axis=1)
        assert rel_l2(out[r_sel][:, heads], o_n[at]) <= 5e-3, f"member {m} out"
        assert lse_err(lse[heads][:, r_sel], l_n[:, at]) <= 1e-3, f"member {m} lse"
        o_full = np.zeros((R, cfg.n_q_heads, cfg.head_dim_v))
        l_full = np.zeros((cfg.n_q_heads, R))
        o_full[np.ix_(need, heads)] = o_n
        l_full[np.ix_(heads, need)] = l_n
        dq_ref, dk_ref, dv_ref = _par.dense_bwd(
            hh, rows=dq_sel, resp_keys=cfg.prefix_len + key_off, out=o_full, lse=l_full,
            kv_heads=None if kv_head is None else kvh, **kw)
        if dq_sel.size:
            assert rel_l2(host(dq)[dq_sel][:, heads], dq_ref) <= 1e-2, f"member {m} dq"
        assert rel_l2(host(dk)[key_off][:, kvh], dk_ref) <= 1e-2, f"member {m} dk"
        assert rel_l2(host(dv)[key_off][:, kvh], dv_ref) <= 1e-2, f"member {m} dv"
        # the prefix pages and the table's prefix entries were never written
        assert torch.equal(prefix.k_pool.index_select(0, pp), k_snap), "prefix K pages written"
        assert torch.equal(prefix.v_pool.index_select(0, pp), v_snap), "prefix V pages written"
        assert torch.equal(prefix.table[:cfg.n_prefix_pages], t_snap), "prefix table entries written"


def test_blockwise_two_members_scaled():
    cfg = configs.C4.scaled(name="c4_scaled", prefix_len=65536, resp_len=2048, block=512,
                            members=2, n_shards=4)
    run_members(cfg, members=[0, 1])


@pytest.mark.timeout(900)
def test_blockwise_c4_block_geometry():
    """c4's response geometry (8,192 tokens in four reverse blocks of 2,048
    rows, 16q/2kv, 256-position pages in a sampled pool with free pages) over a
    16,384-position prefix: every response key's dK/dV, accumulated across the
    blocks (a key of block b is also reached by the rows of every later block),
    and every row's out and lse; dq on 512 rows including each block's first
    and last."""
    cfg = configs.C4.scaled(name="c4_block_geometry", prefix_len=16384, members=1, n_shards=2)
    R, b = cfg.resp_len, cfg.block
    dq_rows = sorted(set(np.random.default_rng(41).choice(R, 504, replace=False).tolist())
                     | {k * b for k in range(R // b)} | {k * b + b - 1 for k in range(R // b)})
    run_members(cfg, members=[0], dq_rows=dq_rows)


@pytest.mark.timeout(1200)
def test_c4_full_size_sampled():
    """c4 at full size: in each of the four 2,048-token blocks, both sides of
    the block edge and of the dq (16-token) and forward (32-token) workgroup
    boundaries at its start, middle and end (48 rows), and the last two response
    keys (test_c4_key_across_blocks covers a key reached by two blocks)."""
    cfg = configs.C4
    R = cfg.resp_len
    rows = sorted({b + o for b in range(0, R, cfg.rows_per_call)
                   for o in (0, 1, 15, 16, 31, 32, 1023, 1024, 2015, 2016, 2046, 2047)
                   if b + o < R})
    run_members(cfg, members=[0], rows=rows, keys=[R - 2, R - 1])


@pytest.mark.timeout(1200)
def test_c4_key_across_blocks():
    """c4 at full size: response key 6,143, the last of block 2, is seen by its
    own row and by every row of block 3, so its dK/dV add up the contributions
    of two block launches.  Checked on KV head 0 and its group's eight query
    heads (the oracle's forward over the 4.46M prefix for those 2,049 rows is
    ~75 TFLOP of fp64): those rows' out and lse and the key's dK/dV."""
    cfg = configs.C4
    key = 3 * cfg.rows_per_call - 1
    run_members(cfg, members=[0], rows=[key, key + 1, cfg.resp_len - 1], keys=[key], dq_rows=[],
                kv_head=0)
