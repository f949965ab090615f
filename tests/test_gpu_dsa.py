"""DSA index selection on the HIP path (needs an MI355X): index scores
(Eq. dsa-index) against the fp64 oracle, and the deterministic top-k
(Eq. glm-global-dsa).

Bars: scores within 2e-6 of the oracle relative to the sum of the terms'
magnitudes (fp32 sums of exact bf16 products); the top-k of the GPU's fp32
scores equals the oracle's top-k of the same scores exactly (the selection
is integer work, decided in the kernel's precision); a merge of per-shard
candidates equals the global selection exactly; against the fp64 scores the
selection is valid: no unselected position scores above a selected one by
more than the score tolerance."""
from __future__ import annotations

import numpy as np
import pytest

import oracle as O
from paper_2607_14952_amd import binding as B
from paper_2607_14952_amd import inputs
from paper_2607_14952_amd.replay import to_device
from tests._gpu import announce, host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu_ready():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()


def _inputs(seed, n_q, H, n_pos, S=64):
    h = inputs.dsa_index_inputs(seed, n_q, H, n_pos, S)
    return h, {k: to_device(v) for k, v in h.items()}


def _term_scale(h, S, b, e):
    """sum_j |w_j| |q_j . k_s| per (row, position): the scale of the fp32 sums."""
    K = O.decode(O.gather(h["k_index_pool"], h["page_table"], S, np.arange(b, e)))
    Q = O.decode(h["q_index"])
    return np.einsum("rh,rhn->rn", np.abs(h["w_index"].astype(np.float64)),
                     np.abs(np.einsum("rhd,nd->rhn", Q, K)))


@pytest.mark.parametrize("H,n_q,rng", [(32, 70, (0, 20000 + 17)), (8, 33, (4096, 9000)),
                                       (16, 32, (0, 64)), (24, 5, (8192, 8192 + 8192 + 31))])
def test_index_scores(H, n_q, rng):
    import torch
    S = 64
    b, e = rng
    h, dev = _inputs(41 + H, n_q, H, e + 100, S)
    announce(f"dsa scores H={H} n_q={n_q} [{b},{e})")
    sc = B.dsa_index_scores(dev["q_index"], dev["w_index"], dev["k_index_pool"],
                            dev["page_table"], pos_begin=b, pos_end=e)
    torch.cuda.synchronize()
    got = host(sc)
    ref = O.dsa_index_scores(h["q_index"], h["w_index"], h["k_index_pool"], h["page_table"],
                             page_size=S, pos_begin=b, pos_end=e)
    scale = _term_scale(h, S, b, e)
    err = np.abs(got - ref) / (scale + 1e-30)
    assert err.max() <= 2e-6, f"max scaled error {err.max():.2e}"


def _gpu_scores(seed=51, n_q=40, H=32, n_pos=30000, S=64):
    h, dev = _inputs(seed, n_q, H, n_pos, S)
    sc = B.dsa_index_scores(dev["q_index"], dev["w_index"], dev["k_index_pool"],
                            dev["page_table"], pos_begin=0, pos_end=n_pos)
    return h, sc


@pytest.mark.parametrize("k,quant", [(2048, None), (100, 0.25), (1, None), (777, 4.0)])
def test_topk_exact_on_gpu_scores(k, quant):
    """The kernel's selection equals the oracle's rule applied to the same
    fp32 scores; quantized scores give heavy ties (lower position first)."""
    import torch
    h, sc = _gpu_scores()
    if quant is not None:
        sc = torch.round(sc / quant) * quant          # many equal scores
    sc = sc.contiguous()
    announce(f"topk k={k} quant={quant}")
    pos, val = B.topk_select(sc, k)
    torch.cuda.synchronize()
    s_host = host(sc)
    want = O.topk_select(s_host.astype(np.float64), k)
    assert np.array_equal(host(pos), want)
    assert np.array_equal(host(val), np.take_along_axis(s_host, want, axis=1))


def test_topk_many_ties_fallback():
    """More than 4,096 keys in the threshold's 12-bit bin (here ~20,000 equal
    scores) take the kernel's full-row radix path; the result still follows the
    rule exactly (lower positions first among the equal scores)."""
    import torch
    g = torch.Generator(device="cuda").manual_seed(7)
    sc = torch.zeros((6, 24000), device="cuda")
    hi = torch.randint(0, 24000, (6, 300), device="cuda", generator=g)
    sc.scatter_(1, hi, torch.rand((6, 300), device="cuda", generator=g) + 1.0)
    sc[:, 5000:5010] = -1.0
    for k in (500, 2048, 23995):
        announce(f"topk ties k={k}")
        pos, _ = B.topk_select(sc, k)
        torch.cuda.synchronize()
        want = O.topk_select(host(sc), k)
        assert np.array_equal(host(pos), want), f"k={k}"


def _check_topk(sc, k, what):
    import torch
    announce(f"topk {what} k={k} shape={tuple(sc.shape)}")
    pos, val = B.topk_select(sc, k)
    torch.cuda.synchronize()
    s_host = host(sc)
    want = O.topk_select(s_host.astype(np.float64), k)
    assert np.array_equal(host(pos), want), what
    assert np.array_equal(host(val).view(np.uint32),
                          np.take_along_axis(s_host, want, axis=1).view(np.uint32)), what


@pytest.mark.parametrize("k", [1, 64, 1000, 2048, 4096])
def test_topk_sampled_bound_path(k):
    """Rows of at least 65,536 keys with k <= 2,048 take the sampled-bound path
    (one pass over the row); k = 4,096 takes the full-row passes.  The
    selection follows the rule exactly either way."""
    import torch
    g = torch.Generator(device="cuda").manual_seed(100 + k)
    _check_topk(torch.randn((5, 200000), device="cuda", generator=g), k, "sampled bound")


def test_topk_sampled_bound_ties():
    """Scores quantized to quarter steps: thousands of keys equal the
    threshold, which the sampled-bound path resolves by lower position."""
    import torch
    g = torch.Generator(device="cuda").manual_seed(11)
    sc = torch.round(torch.randn((4, 131072), device="cuda", generator=g) * 4) / 4
    for k in (1024, 2048):
        _check_topk(sc, k, "sampled ties")


def test_topk_sampled_bound_fallbacks():
    """The exact full-row passes take over (same result) when (a) the sampled
    bound lies too high: the sample blocks hold log-uniform large values that
    the rest of the row never reaches, so fewer than k keys clear the bound;
    (b) one wave's segment holds more candidates than its LDS region (every
    large key in the first eighth of the row); (c) rows are not 16-byte
    aligned (odd leading dimension); (d) every key is equal, so the regions
    overflow and the full-row passes meet more than 4,096 ties in one bin."""
    import torch
    g = torch.Generator(device="cuda").manual_seed(12)
    n = 131072
    sc = torch.randn((3, n), device="cuda", generator=g)
    # sample blocks of a 131,072-key row: 64 blocks of 256 keys at 2,048 j
    blocks = (torch.arange(64, device="cuda")[:, None] * 2048 +
              torch.arange(256, device="cuda")[None, :]).reshape(-1)
    sc[:, blocks] = torch.exp2(torch.rand((3, blocks.numel()), device="cuda", generator=g) * 20)
    _check_topk(sc, 2048, "bound too high")
    sc = torch.randn((3, n), device="cuda", generator=g)
    sc[:, : n // 8] += 10.0
    _check_topk(sc, 2048, "region overflow")
    sc = torch.randn((3, n + 1), device="cuda", generator=g)[:, :n]   # leading dimension n + 1
    _check_topk(sc, 2048, "unaligned rows")
    # every key equal (then one larger key): the regions overflow and the
    # fallback takes its heavy-tie passes; the lowest positions win the ties
    sc = torch.zeros((2, n), device="cuda")
    sc[1, 70000] = 1.0
    _check_topk(sc, 2048, "all equal")


def test_topk_fewer_than_k_and_offsets():
    import torch
    sc = torch.tensor([[1.0, 3.0, 2.0, 3.0, -1.0], [0.0, 0.0, 0.0, 0.0, 0.0]], device="cuda")
    pos, val = B.topk_select(sc, 8, pos_offset=100)
    torch.cuda.synchronize()
    assert host(pos).tolist() == [[100, 101, 102, 103, 104, -1, -1, -1]] * 2
    assert np.all(np.isneginf(host(val)[:, 5:]))
    pos, _ = B.topk_select(sc, 3, pos_offset=100)
    assert host(pos).tolist() == [[101, 102, 103], [100, 101, 102]]


def test_candidate_merge_equals_global():
    """Eq. glm-global-dsa: each contiguous shard's local top-k with global
    positions, concatenated in shard order and merged by the same kernel, is
    the global top-k; one shard's local selection is not."""
    import torch
    h, sc = _gpu_scores(seed=52, n_pos=40000)
    sc = (torch.round(sc * 8) / 8).contiguous()      # ties across shard borders too
    k = 512
    glob, _ = B.topk_select(sc, k)
    bounds = [0, 4096, 13000, 13001, 29999, 40000]
    cps, css = [], []
    for b, e in zip(bounds[:-1], bounds[1:]):
        announce(f"local topk [{b},{e})")
        p, v = B.topk_select(sc[:, b:], k, n=e - b, pos_offset=b)
        keep = min(k, e - b)
        cps.append(p[:, :keep])
        css.append(v[:, :keep])
    cand_pos = torch.cat(cps, dim=1).contiguous()
    cand_sc = torch.cat(css, dim=1).contiguous()
    merged, _ = B.topk_select(cand_sc, k, positions=cand_pos)
    torch.cuda.synchronize()
    assert np.array_equal(host(merged), host(glob))
    assert not np.array_equal(host(cps[0][:, :k]), host(glob))


def test_selection_valid_against_fp64_scores():
    """Against the oracle's fp64 scores, the GPU's top-2048 is a valid top-2048
    up to the score tolerance: min selected >= max unselected - tol."""
    import torch
    h, sc = _gpu_scores(seed=53, n_q=20, n_pos=50000)
    pos, _ = B.topk_select(sc, 2048)
    torch.cuda.synchronize()
    ref = O.dsa_index_scores(h["q_index"], h["w_index"], h["k_index_pool"], h["page_table"],
                             page_size=64, pos_begin=0, pos_end=50000)
    scale = _term_scale(h, 64, 0, 50000)
    tol = 2e-6 * scale.max(axis=1)
    sel = pos.cpu().numpy().astype(np.int64)
    for r in range(ref.shape[0]):
        mask = np.zeros(50000, bool)
        mask[sel[r]] = True
        assert ref[r][mask].min() >= ref[r][~mask].max() - 2 * tol[r]


def test_sparse_replay_with_selection():
    """c5's indices produced by the selection instead of seeded: the global and
    the per-shard-candidate modes give identical indices, equal to the
    oracle's top-k of the GPU scores, and the sparse replay over them matches
    the oracle over the same indices."""
    import torch
    from paper_2607_14952_amd import configs
    from paper_2607_14952_amd.dsa import DsaSelect
    cfg = configs.C5.scaled(name="c5_small_dsa", prefix_len=16384, resp_len=40, topk=300,
                            index_heads=32)
    h = inputs.sparse_inputs(cfg)
    dev = {k: to_device(v) for k, v in h.items()}
    announce(f"dsa select {cfg.name}")
    g = DsaSelect(cfg, dev, mode="global")
    idx = g.run().clone()
    c = DsaSelect(cfg, dev, mode="candidates", n_shards=8)
    idx_c = c.run()
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy(), idx_c.cpu().numpy())
    sc = g.scores[:, :cfg.prefix_len].cpu().numpy().astype(np.float64)
    want = O.topk_select(sc, cfg.topk)
    assert np.array_equal(idx.cpu().numpy(), want)
    # sparse replay over the selected indices vs the oracle over the same indices
    h_sel = dict(h, idx=idx.cpu().numpy())
    from tests.test_gpu_sparse import run as sparse_run
    sparse_run(cfg, h_sel)


@pytest.mark.timeout(900)
def test_dsa_c5_full_size_sampled():
    """c5's selection at full size (2,048 tokens x 2,097,152 positions, 32
    index heads, top-2,048; the sampled-bound top-k path on real index
    scores): sampled rows' scores against the fp64 oracle, their selection
    equal to the oracle's rule on the GPU scores and valid against the fp64
    scores, and the per-shard candidate mode equal to the global one."""
    import torch
    from paper_2607_14952_amd import configs
    from paper_2607_14952_amd.dsa import DsaSelect
    cfg = configs.C5.scaled(index_heads=32)
    announce("dsa c5: inputs")
    h = inputs.sparse_inputs(cfg)
    dev = {k: to_device(h[k]) for k in ("q_index", "w_index", "k_index_pool", "page_table")}
    announce("dsa c5: global selection")
    g = DsaSelect(cfg, dev, mode="global")
    idx = g.run().clone()
    announce("dsa c5: candidate selection")
    idx_c = DsaSelect(cfg, dev, mode="candidates", n_shards=8).run()
    torch.cuda.synchronize()
    assert np.array_equal(host(idx), host(idx_c)), "candidates == global"
    rows = [0, 1, 1000, cfg.resp_len - 1]
    P = cfg.prefix_len
    sc = host(g.scores[rows, :P])
    want = O.topk_select(sc.astype(np.float64), cfg.topk)
    assert np.array_equal(host(idx)[rows], want), "selection == the rule on the GPU scores"
    announce("dsa c5: oracle scores for the sampled rows")
    hr = dict(h, q_index=h["q_index"][rows], w_index=h["w_index"][rows])
    ref = O.dsa_index_scores(hr["q_index"], hr["w_index"], h["k_index_pool"], h["page_table"],
                             page_size=cfg.page_size, pos_begin=0, pos_end=P)
    # sum_j |w_j| |q_j . k_s| per row, with matrix products (2M positions)
    K = O.decode(O.gather(h["k_index_pool"], h["page_table"], cfg.page_size, np.arange(P)))
    scale = np.stack([np.abs(hr["w_index"][j].astype(np.float64)) @
                      np.abs(O.decode(hr["q_index"][j]) @ K.T) for j in range(len(rows))])
    del K
    err = np.abs(sc - ref) / np.maximum(scale, 1e-30)
    assert err.max() <= 2e-6, f"max scaled error {err.max():.2e}"
    tol = 2e-6 * scale.max(axis=1)
    for j in range(len(rows)):
        mask = np.zeros(P, bool)
        mask[want[j]] = True
        assert ref[j][mask].min() >= ref[j][~mask].max() - 2 * tol[j], f"row {rows[j]}"
