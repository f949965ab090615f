"""The thread-pool oracle helpers of the full-size parity tests compose key
ranges and row chunks back into the unsplit oracle result (CPU only)."""
import numpy as np

import oracle as O
from tests import _par
from tests._tiny import make, rel_l2


def test_dense_ranges_compose_to_the_unsplit_oracle():
    t = make(P=300, R=9, Hq=4, Hkv=2, D=8, S=16, seed=31)
    h = dict(q=t.q, k_pool=t.k_pool, v_pool=t.v_pool, page_table=t.page_table, d_out=t.d_out)
    kw = dict(page_size=t.S, q_pos0=t.P, scale=t.scale)
    rows = np.array([0, 3, 4, 8])
    o, lse = _par.dense_fwd(h, rows=rows, prefix_len=t.P, piece=64, **kw)
    o_ref, l_ref = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, rows=rows, **kw)
    assert rel_l2(o, o_ref) < 1e-12 and np.max(np.abs(lse - l_ref)) < 1e-12
    o_all, l_all = _par.dense_fwd(h, rows=np.arange(t.R), prefix_len=t.P, piece=64, **kw)
    keys = np.array([t.P + 2, t.P + 7])
    dq, dk, dv = _par.dense_bwd(h, prefix_len=t.P, rows=rows, resp_keys=keys, out=o_all,
                                lse=l_all, piece=64, resp_piece=4, **kw)
    dq_ref, dk_ref, dv_ref = O.attn_bwd(t.q, t.k_pool, t.v_pool, t.page_table, t.d_out,
                                        prefix_len=t.P, rows=rows, resp_keys=keys, **kw)
    for a, b in ((dq, dq_ref), (dk, dk_ref), (dv, dv_ref)):
        assert rel_l2(a, b) < 1e-12
    # one KV head's group: out/lse of its query heads, its dq heads and dK/dV
    o1, l1 = _par.dense_fwd(h, rows=rows, prefix_len=t.P, piece=64, heads=[2, 3], **kw)
    assert rel_l2(o1, o_ref[:, [2, 3]]) < 1e-12 and np.max(np.abs(l1 - l_ref[[2, 3]])) < 1e-12
    dq1, dk1, dv1 = _par.dense_bwd(h, prefix_len=t.P, rows=rows, resp_keys=keys, out=o_all,
                                   lse=l_all, piece=64, resp_piece=4, kv_heads=[1], **kw)
    for a, b in ((dq1, dq_ref[:, [2, 3]]), (dk1, dk_ref[:, [1]]), (dv1, dv_ref[:, [1]])):
        assert rel_l2(a, b) < 1e-12


def test_sparse_row_chunks_compose():
    t = make(P=40, R=7, Hq=3, Hkv=1, D=6, S=4, seed=32)
    rng = np.random.default_rng(3)
    idx = np.stack([np.sort(rng.choice(t.P, 9, replace=False)) for _ in range(t.R)]).astype(np.int32)
    d_out = t.d_out[..., :4]
    h = dict(q=t.q, latent_pool=t.k_pool, page_table=t.page_table, idx=idx, d_out=d_out)
    kw = dict(page_size=t.S, prefix_len=t.P, q_pos0=t.P, scale=t.scale)
    rows = np.array([0, 2, 3, 6])
    o, lse, dq = _par.sparse(h, rows=rows, head_dim_v=4, **kw)
    o_ref, l_ref = O.sparse_fwd(t.q, t.k_pool, t.page_table, idx, head_dim_v=4, rows=rows, **kw)
    dq_ref = O.sparse_bwd(t.q, t.k_pool, t.page_table, idx, d_out, head_dim_v=4, rows=rows, **kw)
    assert rel_l2(o, o_ref) < 1e-13 and np.max(np.abs(lse - l_ref)) < 1e-13
    assert rel_l2(dq, dq_ref) < 1e-13
