"""Blockwise replay against a resident prefix (append -> reverse blocks -> pop)
vs the fp64 oracle of the unblocked response (needs an MI355X)."""
from __future__ import annotations

import numpy as np
import pytest

import oracle as O
from paper_2607_14952_amd import binding as B
from paper_2607_14952_amd import configs, inputs
from paper_2607_14952_amd.blockwise import BlockwiseReplay, ResidentPrefix
from paper_2607_14952_amd.replay import to_device
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


def run_members(cfg, members, rows=None, keys=None):
    import torch
    store = inputs.prefix_store(cfg)
    prefix = ResidentPrefix(cfg, store)
    rep = BlockwiseReplay(cfg, prefix)
    for m in members:
        resp = inputs.response_inputs(cfg, m)
        dev = {k: to_device(v) for k, v in resp.items()}
        pages = prefix.free[:cfg.n_resp_pages]
        keep = {}
        announce(f"{cfg.name} member {m}")
        dq, dk, dv = rep.run_member(dev, keep=keep)
        torch.cuda.synchronize()
        kp, vp, table = logical_store(cfg, store, resp, pages)
        kw = dict(page_size=cfg.page_size, q_pos0=cfg.prefix_len, scale=cfg.scale)
        r_sel = np.arange(cfg.resp_len) if rows is None else np.asarray(rows)
        o_ref, l_ref = O.attn_fwd(resp["q"], kp, vp, table, rows=r_sel, **kw)
        out = np.concatenate([host(keep[b][0]) for b in range(cfg.blocks)])
        lse = np.concatenate([host(keep[b][1]) for b in range(cfg.blocks)], axis=1)
        assert rel_l2(out[r_sel], o_ref) <= 5e-3, f"member {m} out"
        assert lse_err(lse[:, r_sel], l_ref) <= 1e-3, f"member {m} lse"
        o_full = np.zeros((cfg.resp_len, cfg.n_q_heads, cfg.head_dim_v))
        l_full = np.zeros((cfg.n_q_heads, cfg.resp_len))
        need = r_sel if keys is None else np.union1d(r_sel, np.arange(min(keys) - cfg.prefix_len, cfg.resp_len))
        o_n, l_n = (o_ref, l_ref) if need is r_sel else O.attn_fwd(resp["q"], kp, vp, table, rows=need, **kw)
        o_full[need], l_full[:, need] = o_n, l_n
        dq_ref, dk_ref, dv_ref = O.attn_bwd(resp["q"], kp, vp, table, resp["d_out"], rows=r_sel,
                                            resp_keys=keys, out=o_full, lse=l_full,
                                            prefix_len=cfg.prefix_len, **kw)
        k_rows = (np.arange(cfg.resp_len) if keys is None else np.asarray(keys) - cfg.prefix_len)
        assert rel_l2(host(dq)[r_sel], dq_ref) <= 1e-2, f"member {m} dq"
        assert rel_l2(host(dk)[k_rows], dk_ref) <= 1e-2, f"member {m} dk"
        assert rel_l2(host(dv)[k_rows], dv_ref) <= 1e-2, f"member {m} dv"
    # the prefix pages were never written
    assert np.array_equal(prefix.table_host[:cfg.n_prefix_pages], store["prefix_table"])


def test_blockwise_two_members_scaled():
    cfg = configs.C4.scaled(name="c4_scaled", prefix_len=65536, resp_len=2048, block=512,
                            members=2, n_shards=4)
    run_members(cfg, members=[0, 1])


@pytest.mark.timeout(1200)
def test_c4_full_size_sampled():
    cfg = configs.C4
    R = cfg.resp_len
    rows = [0, 2047, 2048, 6000, R - 1]
    keys = [cfg.prefix_len + R - 2, cfg.prefix_len + R - 1]
    run_members(cfg, members=[0], rows=rows, keys=keys)
