"""The FLOP convention that every TFLOP/s figure of the benchmark divides by
(CPU).  Each count is checked against an independent product written out from
the workload's shape, and against the totals stated for the workloads:

* dense replay, per visible (row, key) pair and query head: the forward runs
  Q.K^T and P.V (2 D-wide contractions, 2 FLOP each); the backward recomputes
  Q.K^T and forms dO.V^T and dS.K for every key, plus dS^T.Q and P^T.dO for the
  response keys, whose dK/dV are produced (Sec. "Response Replay": prefix
  entries get no gradient);
* blockwise replay: the same counts per block, rows of block b attending to the
  prefix and causally to the response up to themselves;
* sparse latent replay: Dk-wide Q.K^T and Dv-wide P.V forward; the dq-only
  backward recomputes Q.K^T and forms dO.V^T and dS.K.
"""
from __future__ import annotations

import pytest

import bench
from paper_2607_14952_amd import configs
from paper_2607_14952_amd.blockwise import block_flops


def _pairs(R, P):
    """(prefix pairs, response pairs) by direct count of visible (row, key)."""
    pre = R * P
    resp = 0
    for i in range(R):
        resp += i + 1
    return pre, resp


def test_visible_counts_brute_force():
    for R, P in ((1, 0), (1, 5), (7, 13), (128, 4096)):
        cfg = configs.C1.__class__(**{**configs.C1.__dict__, "resp_len": R, "prefix_len": P})
        assert bench.visible_counts(cfg) == _pairs(R, P)


def test_dense_counts():
    c1_fwd, c1_bwd = bench.flops(configs.C1)
    assert c1_fwd / 1e9 == pytest.approx(0.273, abs=5e-4)
    assert c1_bwd / 1e9 == pytest.approx(0.413, abs=5e-4)
    assert bench.flops(configs.C2)[0] / 1e12 == pytest.approx(17.73, abs=5e-3)
    fwd, bwd = bench.flops(configs.C3)
    assert fwd / 1e12 == pytest.approx(140.87, abs=5e-3)
    assert bwd / 1e12 == pytest.approx(211.45, abs=5e-3)
    assert (fwd + bwd) / 1e12 == pytest.approx(352.32, abs=5e-3)
    # the same numbers from the contraction list
    cfg = configs.C3
    pre, resp = _pairs(cfg.resp_len, cfg.prefix_len)
    per_pair = 2 * cfg.n_q_heads * cfg.head_dim
    assert fwd == per_pair * 2 * (pre + resp)
    assert bwd == per_pair * (3 * pre + 5 * resp)
    # work that the replay actually needs, without the Q.K^T recompute
    assert bench.useful_flops(cfg) == per_pair * (4 * pre + 6 * resp)


def test_blockwise_counts():
    cfg = configs.C4
    blocks = [block_flops(cfg, b) for b in range(cfg.blocks)]
    assert len(blocks) == 4
    for f, b in blocks:                    # the stated ranges are to one decimal
        assert 149.6 <= round(f / 1e12, 1) <= 149.8
        assert 224.4 <= round(b / 1e12, 1) <= 224.9
    member = sum(f + b for f, b in blocks)
    assert member / 1e12 == pytest.approx(1497.3, abs=0.05)
    assert member * cfg.members / 1e15 == pytest.approx(11.98, abs=5e-3)
    # the blocks partition the member: same total as one call over all rows
    whole = bench.flops(cfg)
    assert member == sum(whole)


def test_sparse_counts():
    cfg = configs.C5
    fwd, bwd = bench.sparse_flops(cfg)
    assert fwd / 1e12 == pytest.approx(1.753, abs=5e-4)
    assert bwd / 1e12 == pytest.approx(2.680, abs=1e-3)
    vis = cfg.resp_len * cfg.topk + _pairs(cfg.resp_len, 0)[1]
    assert fwd == 2 * cfg.n_q_heads * vis * (576 + 512)
    assert bwd == 2 * cfg.n_q_heads * vis * (576 + 512 + 576)
    # gathered latent rows per pass, one 576-wide bf16 row per selected entry
    # (the stated 4.83 GB); the benchmark's gather rate also counts the causal
    # window's rows, which the kernels read the same way
    assert cfg.resp_len * cfg.topk * 576 * 2 / 1e9 == pytest.approx(4.83, abs=5e-3)
