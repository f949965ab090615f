"""The paper's production composition on the HIP path vs the fp64 oracle
(needs an MI355X): the numerator reduced in bf16 (the note after Eq.
qwen-global-attn) and block-cyclic page ownership (Eq. qwen-page-owner).

Bars: bf16-numerator merge on exact fp32 parts within 2 bf16 ulps of the
largest partial sum the reduction can reach (the sum of the terms' magnitudes)
per element, and identical to the oracle's composition to 1e-6 on at least 99%
of the elements (the two sides form e^(l_r - m) o_r in fp32 and fp64, which may
round a term to a neighbouring bf16 value and shift later partial sums by one
of their ulps); replay bars as in
the dense parity tests (out rel-L2 <= 5e-3, lse max-abs <= 1e-3, grads rel-L2
<= 1e-2)."""
from __future__ import annotations

import numpy as np
import pytest

import oracle as O
from paper_2607_14952_amd import binding as B
from paper_2607_14952_amd import configs, inputs
from paper_2607_14952_amd.replay import ReplayStep, device_inputs
from tests._gpu import TOL_BF16, announce, host, lse_err, rel_l2

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu_ready():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()


@pytest.mark.parametrize("n_parts,n_q", [(9, 37), (2, 1), (33, 130)])
def test_merge_bf16_numerator(n_parts, n_q):
    import torch
    H, Dv = 16, 256
    o, lse = inputs.merge_parts(31 + n_parts, n_parts, n_q, H, Dv)
    announce(f"merge bf16 numerator parts={n_parts} n_q={n_q}")
    out, l_gpu = B.lse_merge(torch.from_numpy(o).cuda(), torch.from_numpy(lse).cuda(),
                             out_dtype=torch.float32, flags=B.FLAG_BF16_NUMERATOR)
    out_f32, l_f32 = B.lse_merge(torch.from_numpy(o).cuda(), torch.from_numpy(lse).cuda(),
                                 out_dtype=torch.float32)
    torch.cuda.synchronize()
    got = host(out)
    want, want_l = O.lse_merge_bf16_numerator(list(o), list(lse))
    exact, _ = O.lse_merge(list(o), list(lse))
    # the largest partial sum each element's reduction can reach (its bf16 ulp scale)
    L = lse.astype(np.float64)
    m = np.max(L, axis=0)
    w = np.where(np.isfinite(L), np.exp(L - np.where(np.isfinite(m), m, 0.0)[None]), 0.0)
    a = np.where(np.isfinite(m), w.sum(0), 1.0)
    big = np.sum(np.abs(np.einsum("shr,srhd->srhd", w, o)), axis=0) / a.T[:, :, None]
    err = np.abs(got - want)
    assert np.all(err <= 4 * 2.0 ** -8 * big + 1e-30), \
        f"max err / scale {np.max(err / (big + 1e-30)):.4f}"
    close = err <= 1e-6 * (np.abs(want) + 1e-30)
    assert close.mean() >= 0.99, f"only {close.mean():.4f} of elements match the oracle"
    assert lse_err(host(l_gpu), want_l) <= 1e-5
    assert np.array_equal(host(l_gpu), host(l_f32)), "lse does not depend on the flag"
    # the flag rounds: its distance to the exact composition is bf16-sized, the fp32 merge's is not
    d_bf16 = np.max(np.abs(got - exact) / (big + 1e-30))
    d_f32 = np.max(np.abs(host(out_f32) - exact) / (big + 1e-30))
    assert d_bf16 > 2.0 ** -14 and d_f32 < 2.0 ** -18, (d_bf16, d_f32)


CYCLIC = configs.C3.scaled(name="cyclic_small", prefix_len=256 * 61 + 100, resp_len=96,
                           n_shards=8, splits_per_shard=2, ownership="cyclic", plant_frac=0.01)


def test_cyclic_ownership_replay():
    """Shards own pages p mod 8 (ragged: 62 pages, the last one partial); the
    composed forward and the summed backward equal the unsharded oracle."""
    import torch
    cfg = CYCLIC
    h = inputs.dense_inputs(cfg)
    dev = device_inputs(h)
    announce(f"cyclic replay {cfg.name}")
    step = ReplayStep(cfg, dev)
    assert len(step.shards) == 9 and step.shards[-1] == (cfg.prefix_len, cfg.kv_len)
    step.step()
    torch.cuda.synchronize()
    kw = dict(page_size=cfg.page_size, q_pos0=cfg.q_pos0, scale=cfg.scale)
    o_ref, l_ref = O.attn_fwd(h["q"], h["k_pool"], h["v_pool"], h["page_table"], **kw)
    assert rel_l2(host(step.out), o_ref) <= TOL_BF16["out"]
    assert lse_err(host(step.lse), l_ref) <= TOL_BF16["lse"]
    # each shard's result is the oracle over exactly its owned positions
    for c in (0, 5, 7):
        pos = O.cyclic_owned_positions(cfg.prefix_len, cfg.page_size, cfg.n_shards, c)
        assert pos.size == cfg.shard_len(c)
        so, sl = O.attn_fwd(h["q"], h["k_pool"], h["v_pool"], h["page_table"],
                            key_positions=pos, **kw)
        assert rel_l2(host(step.shard_out[c]), so) <= TOL_BF16["out"], f"shard {c} out"
        assert lse_err(host(step.shard_lse[c]), sl) <= TOL_BF16["lse"], f"shard {c} lse"
    dq_ref, dk_ref, dv_ref = O.attn_bwd(h["q"], h["k_pool"], h["v_pool"], h["page_table"],
                                        h["d_out"], page_size=cfg.page_size,
                                        prefix_len=cfg.prefix_len, q_pos0=cfg.q_pos0,
                                        scale=cfg.scale, out=o_ref, lse=l_ref)
    assert rel_l2(host(step.dq), dq_ref) <= TOL_BF16["grad"]
    assert rel_l2(host(step.dk), dk_ref) <= TOL_BF16["grad"]
    assert rel_l2(host(step.dv), dv_ref) <= TOL_BF16["grad"]


def test_cyclic_bf16_numerator_forward():
    """With the bf16 numerator the composed output follows the oracle's bf16
    composition of the oracle's shard results (within the kernels' own bar)
    and differs from the fp32 composition by bf16 rounding only."""
    import torch
    cfg = CYCLIC.scaled(name="cyclic_bf16num", bf16_numerator=True, backward=False)
    h = inputs.dense_inputs(cfg, with_dout=False)
    dev = device_inputs(h)
    announce(f"cyclic bf16-numerator forward {cfg.name}")
    step = ReplayStep(cfg, dev)
    step.forward()
    ref32 = ReplayStep(cfg.scaled(bf16_numerator=False), dev)
    ref32.forward()
    torch.cuda.synchronize()
    kw = dict(page_size=cfg.page_size, q_pos0=cfg.q_pos0, scale=cfg.scale)
    parts = [O.attn_fwd(h["q"], h["k_pool"], h["v_pool"], h["page_table"],
                        key_positions=O.cyclic_owned_positions(cfg.prefix_len, cfg.page_size,
                                                               cfg.n_shards, c), **kw)
             for c in range(cfg.n_shards)]
    parts.append(O.attn_fwd(h["q"], h["k_pool"], h["v_pool"], h["page_table"],
                            kv_begin=cfg.prefix_len, kv_end=cfg.kv_len, **kw))
    o_ref, l_ref = O.lse_merge_bf16_numerator([p[0] for p in parts], [p[1] for p in parts])
    assert rel_l2(host(step.out), o_ref) <= TOL_BF16["out"]
    assert lse_err(host(step.lse), l_ref) <= TOL_BF16["lse"]
    assert np.array_equal(host(step.lse), host(ref32.lse)), "lse does not depend on the flag"
    d = np.abs(host(step.out).astype(np.float64) - host(ref32.out).astype(np.float64))
    assert 0 < d.max() <= 4 * 2.0 ** -8 * np.abs(host(ref32.out)).max()
