"""Output canaries: every output and workspace of each entry point sits inside
guard regions filled with a sentinel byte, and after the call (ragged shapes:
one query row, partial row tiles, 16-position pages, unaligned splits, 256
heads, row strides wider than the rows, a top-k longer than its row) the
guards and the gaps between strided rows still hold the sentinel: no kernel
writes outside what its call names (needs an MI355X)."""
from __future__ import annotations

import ctypes

import numpy as np
import pytest

from paper_2607_14952_amd import binding as B
from paper_2607_14952_amd import configs, inputs
from paper_2607_14952_amd.replay import device_inputs, to_device
from tests._gpu import announce

pytestmark = pytest.mark.gpu

SENTINEL = 0xA5
GUARD = 1 << 16


@pytest.fixture(scope="module", autouse=True)
def _gpu_ready():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()


class Guarded:
    """A tensor of `shape` (or `nbytes` of uint8) inside sentinel-filled guards."""

    def __init__(self, shape, dtype, nbytes=None):
        import torch
        esz = torch.empty((), dtype=dtype).element_size()
        self.n = nbytes if nbytes is not None else int(np.prod(shape)) * esz
        pad = -self.n % 256
        self.buf = torch.full((GUARD + self.n + pad + GUARD,), SENTINEL, dtype=torch.uint8,
                              device="cuda")
        body = self.buf[GUARD:GUARD + self.n]
        self.t = body if nbytes is not None else body.view(dtype).view(shape)

    def intact(self):
        b = self.buf
        return bool((b[:GUARD] == SENTINEL).all()) and bool((b[GUARD + self.n:] == SENTINEL).all())


def assert_intact(name, *gs):
    import torch
    torch.cuda.synchronize()
    for i, g in enumerate(gs):
        assert g.intact(), f"{name}: a write landed outside output {i}"


def _dense_case(cfg, splits, ranges):
    import torch
    h = inputs.dense_inputs(cfg)
    dev = device_inputs(h)
    kv = B.PagedKV(dev["k_pool"], dev["v_pool"], dev["page_table"])
    R, Hq, D, Dv, Hkv = cfg.resp_len, cfg.n_q_heads, cfg.head_dim, cfg.head_dim_v, cfg.n_kv_heads
    P, q0 = cfg.prefix_len, cfg.q_pos0
    kw = dict(prefix_len=P, q_pos0=q0, scale=cfg.scale)
    announce(f"canary fwd {cfg.name}")
    op, lp = Guarded((len(splits), R, Hq, Dv), torch.float32), Guarded((len(splits), Hq, R), torch.float32)
    B.prefix_attn_fwd(dev["q"], kv, splits, out_part=op.t, lse_part=lp.t, **kw)
    assert_intact("prefix_attn_fwd", op, lp)
    for bf16_num in (False, True):
        announce(f"canary merge {cfg.name} bf16_numerator={bf16_num}")
        o, l = Guarded((R, Hq, Dv), dev["q"].dtype), Guarded((Hq, R), torch.float32)
        B.lse_merge(op.t, lp.t, out=o.t, lse=l.t, flags=B.FLAG_BF16_NUMERATOR if bf16_num else 0)
        assert_intact("lse_merge", o, l)
    p = B.make_params(dev["q"], kv, **kw)
    need = B.load_library().ls_prefix_attn_bwd_workspace_size(ctypes.byref(p))
    ws = Guarded(None, torch.uint8, nbytes=need)
    dq = Guarded((R, Hq, D), torch.float32)
    dk = Guarded((q0 + R - P, Hkv, D), torch.float32)
    dv = Guarded((q0 + R - P, Hkv, Dv), torch.float32)
    dk.t.zero_()
    dv.t.zero_()
    for r, (b, e) in enumerate(ranges):
        announce(f"canary bwd {cfg.name} range {r}")
        B.prefix_attn_bwd(dev["q"], kv, dev["d_out"], o.t, l.t, kv_begin=b, kv_end=e,
                          flags=(B.FLAG_ACCUMULATE_DQ | B.FLAG_PREP_READY) if r else 0,
                          dq=dq.t, dk_resp=dk.t, dv_resp=dv.t, workspace=ws.t, **kw)
        assert_intact("prefix_attn_bwd", dq, dk, dv, ws)
    announce(f"canary gather {cfg.name}")
    b, e = 3, min(cfg.kv_len, 1111)
    ko = Guarded((e - b, Hkv, D), dev["k_pool"].dtype)
    vo = Guarded((e - b, Hkv, Dv), dev["v_pool"].dtype)
    B.gather_kv(kv, b, e, k_out=ko.t, v_out=vo.t)
    assert_intact("gather_kv", ko, vo)


BASE = configs.C3.scaled(name="canary", prefix_len=4096, resp_len=64, n_shards=2,
                         splits_per_shard=2, plant_frac=0.0)


def test_canaries_dense_single_row():
    cfg = BASE.scaled(name="canary_r1", prefix_len=512, resp_len=1, n_shards=1)
    _dense_case(cfg, [(0, 512), (512, 513)], [(0, 512), (512, 513)])


def test_canaries_dense_page16_partial_tiles():
    cfg = BASE.scaled(name="canary_p16", page_size=16, prefix_len=3000, resp_len=77)
    P = cfg.prefix_len
    _dense_case(cfg, [(0, 1000), (1000, 1003), (1003, P), (P, P + 40), (P + 40, P + 77)],
                [(0, 1234), (1234, P + 50), (P + 50, P + 77)])


def test_canaries_dense_ragged_groups_and_f32():
    cfg = BASE.scaled(name="canary_g2", n_q_heads=6, n_kv_heads=3, prefix_len=2048, resp_len=45)
    _dense_case(cfg, [(0, 2048), (2048, 2093)], [(0, 2048), (2048, 2093)])
    cfg = configs.C1.scaled(name="canary_f32", prefix_len=640, resp_len=33)
    _dense_case(cfg, [(0, 320), (320, 640), (640, 673)], [(0, 640), (640, 673)])
    # 650 tokens x 8 heads = 5,200 packed rows: three dK/dV row chunks, a partial
    # last tile and a partial sixth key block of the dK/dV kernel
    cfg = BASE.scaled(name="canary_dkdv", prefix_len=1024, resp_len=650, n_shards=1)
    _dense_case(cfg, [(0, 1024), (1024, 1674)], [(0, 1024), (1024, 1674)])


def test_canaries_scatter():
    """The scatter writes only the rows the table names for its positions."""
    import torch
    cfg = BASE.scaled(name="canary_scatter", page_size=16, prefix_len=1000, resp_len=77)
    h = inputs.dense_inputs(cfg, with_dout=False)
    dev = device_inputs(h)
    kp = Guarded(tuple(dev["k_pool"].shape), dev["k_pool"].dtype)
    vp = Guarded(tuple(dev["v_pool"].shape), dev["v_pool"].dtype)
    kp.t.copy_(dev["k_pool"])
    vp.t.copy_(dev["v_pool"])
    kv = B.PagedKV(kp.t, vp.t, dev["page_table"])
    b, n = cfg.prefix_len + 5, 61
    src_k = torch.randn((n, cfg.n_kv_heads, 256), device="cuda").to(torch.bfloat16)
    src_v = torch.randn((n, cfg.n_kv_heads, 256), device="cuda").to(torch.bfloat16)
    announce("canary scatter")
    B.scatter_kv(kv, b, src_k, src_v)
    assert_intact("scatter_kv", kp, vp)
    table = h["page_table"]
    j = np.arange(b, b + n)
    page, slot = table[j // cfg.page_size], j % cfg.page_size
    mask = torch.ones(dev["k_pool"].shape[:2], dtype=torch.bool, device="cuda")
    mask[torch.from_numpy(page.astype(np.int64)), torch.from_numpy(slot.astype(np.int64))] = False
    assert torch.equal(kp.t[mask], dev["k_pool"][mask]) and torch.equal(vp.t[mask], dev["v_pool"][mask])
    assert torch.equal(kp.t[torch.from_numpy(page.astype(np.int64)), torch.from_numpy(slot.astype(np.int64))], src_k)


@pytest.mark.parametrize("heads,R,topk", [(256, 23, 97), (128, 1, 64)])
def test_canaries_sparse(heads, R, topk):
    import torch
    cfg = configs.C5.scaled(name=f"canary_sparse_{heads}_{R}", prefix_len=8192, resp_len=R,
                            topk=topk, n_q_heads=heads)
    h = inputs.sparse_inputs(cfg)
    q = to_device(h["q"])
    lat = to_device(h["latent_pool"])
    kv = B.PagedKV(lat, lat, to_device(h["page_table"]))
    idx = to_device(h["idx"])
    kw = dict(prefix_len=cfg.prefix_len, q_pos0=cfg.q_pos0, scale=cfg.scale)
    lib = B.load_library()
    p = B._sparse_params(q, kv, **kw)
    o, l = Guarded((R, heads, 512), torch.float32), Guarded((heads, R), torch.float32)
    wf = Guarded(None, torch.uint8, nbytes=lib.ls_sparse_attn_workspace_size(ctypes.byref(p), topk, 0))
    announce(f"canary sparse fwd {heads} {R}")
    B.sparse_attn_fwd(q, kv, idx, out=o.t, lse=l.t, workspace=wf.t, **kw)
    assert_intact("sparse_attn_fwd", o, l, wf)
    o2, l2 = Guarded((R, heads, 512), torch.float32), Guarded((heads, R), torch.float32)
    announce(f"canary sparse fwd noalloc {heads} {R}")
    B.sparse_attn_fwd_noalloc(q, kv, idx, out=o2.t, lse=l2.t, **kw)
    assert_intact("sparse_attn_fwd_noalloc", o2, l2)
    dq = Guarded((R, heads, 576), torch.float32)
    wb = Guarded(None, torch.uint8, nbytes=lib.ls_sparse_attn_workspace_size(ctypes.byref(p), topk, 1))
    announce(f"canary sparse bwd {heads} {R}")
    B.sparse_attn_bwd(q, kv, idx, to_device(h["d_out"]), o.t.to(torch.bfloat16), l.t, dq=dq.t,
                      workspace=wb.t, **kw)
    assert_intact("sparse_attn_bwd", dq, wb)


def test_canaries_dsa_scores_and_topk():
    """Scores written into rows of a wider array (ld > n) and a top-k longer
    than its rows (n < k, pads) into rows of a wider array (out_ld > k): the
    gap columns keep the sentinel."""
    import torch
    n_q, H, S = 5, 24, 64
    b, e = 32, 32 + 1000
    h = inputs.dsa_index_inputs(61, n_q, H, e + 64, S)
    dev = {k: to_device(v) for k, v in h.items()}
    ld = 1012
    sc = Guarded((n_q, ld), torch.float32)
    announce("canary dsa scores")
    B.dsa_index_scores(dev["q_index"], dev["w_index"], dev["k_index_pool"], dev["page_table"],
                       pos_begin=b, pos_end=e, scores=sc.t)
    assert_intact("dsa_index_scores", sc)
    gap = sc.t[:, e - b:].contiguous().view(torch.uint8)
    assert bool((gap == SENTINEL).all()), "dsa_index_scores wrote past a row's positions"
    k, n, out_ld = 128, 100, 136
    op = Guarded((n_q, out_ld), torch.int32)
    os_ = Guarded((n_q, out_ld), torch.float32)
    announce("canary top-k")
    B.topk_select(sc.t[:, :n], k, n=n, out_pos=op.t[:, :k], out_scores=os_.t[:, :k])
    assert_intact("topk_select", op, os_)
    for t in (op.t, os_.t):
        assert bool((t[:, k:].contiguous().view(torch.uint8) == SENTINEL).all()), \
            "topk_select wrote past k"
    assert bool((op.t[:, n:k] == -1).all())


def test_canaries_read_probe():
    import torch
    buf = torch.ones(1 << 20, dtype=torch.float32, device="cuda")
    out = Guarded((1,), torch.int32)
    announce("canary read probe")
    B.hbm_read_probe(buf, out.t)
    assert_intact("hbm_read_probe", out)
