"""HIP path vs the fp64 oracle on identical seeded inputs (needs an MI355X).

Every call goes through the C ABI (ctypes binding); the oracle never sees a
value the GPU produced.  Bars: bit-exact for the page gather; bf16 inputs:
out rel-L2 <= 5e-3, lse max-abs <= 1e-3, dq/dk/dv rel-L2 <= 1e-2; fp32 inputs:
rel-L2 <= 1e-5 and lse max-abs <= 1e-5.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle as O
from paper_2607_14952_amd import binding as B
from paper_2607_14952_amd import configs, inputs
from paper_2607_14952_amd.replay import ReplayStep, device_inputs
from tests import _par
from tests._gpu import announce, host, lse_err, oracle_bkw, oracle_kw, rel_l2, tol

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu_ready():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()


def _kv(dev, epoch=0):
    return B.PagedKV(dev["k_pool"], dev["v_pool"], dev["page_table"], epoch)


def check_forward(cfg, h, dev, splits, *, P, q_pos0):
    """Per-split (o_r, l_r) and the merged (o, l) against the oracle."""
    t = tol(cfg)
    kv = _kv(dev)
    announce(f"fwd {cfg.name} R={h['q'].shape[0]} splits={len(splits)} q_pos0={q_pos0}")
    o_part, l_part = B.prefix_attn_fwd(dev["q"], kv, splits, prefix_len=P, q_pos0=q_pos0,
                                       scale=cfg.scale)
    out, lse = B.lse_merge(o_part, l_part, out_dtype=dev["q"].dtype)
    import torch
    torch.cuda.synchronize()
    kw = dict(page_size=cfg.page_size, q_pos0=q_pos0, scale=cfg.scale)
    for s, (b, e) in enumerate(splits):
        o_ref, l_ref = O.attn_fwd(h["q"], h["k_pool"], h["v_pool"], h["page_table"],
                                  kv_begin=b, kv_end=e, **kw)
        assert rel_l2(host(o_part[s]), o_ref) <= t["out"], f"split {s} out"
        assert lse_err(host(l_part[s]), l_ref) <= t["lse"], f"split {s} lse"
    o_ref, l_ref = O.attn_fwd(h["q"], h["k_pool"], h["v_pool"], h["page_table"], **kw)
    err_o, err_l = rel_l2(host(out), o_ref), lse_err(host(lse), l_ref)
    assert err_o <= t["out"], f"merged out rel-L2 {err_o:.2e}"
    assert err_l <= t["lse"], f"merged lse max-abs {err_l:.2e}"
    return out, lse, o_ref, l_ref


def check_backward(cfg, h, dev, out, lse, o_ref, l_ref, ranges, *, P, q_pos0):
    t = tol(cfg)
    kv = _kv(dev)
    dq = dk = dv = None
    announce(f"bwd {cfg.name} ranges={len(ranges)}")
    for r, (b, e) in enumerate(ranges):
        dq, dk, dv = B.prefix_attn_bwd(dev["q"], kv, dev["d_out"], out, lse, prefix_len=P,
                                       q_pos0=q_pos0, scale=cfg.scale, kv_begin=b, kv_end=e,
                                       flags=B.FLAG_ACCUMULATE_DQ if r else 0, dq=dq, dk_resp=dk,
                                       dv_resp=dv)
    import torch
    torch.cuda.synchronize()
    dq_ref, dk_ref, dv_ref = O.attn_bwd(h["q"], h["k_pool"], h["v_pool"], h["page_table"],
                                        h["d_out"], page_size=cfg.page_size, prefix_len=P,
                                        q_pos0=q_pos0, scale=cfg.scale, out=o_ref, lse=l_ref)
    e_q, e_k, e_v = rel_l2(host(dq), dq_ref), rel_l2(host(dk), dk_ref), rel_l2(host(dv), dv_ref)
    assert e_q <= t["grad"], f"dq rel-L2 {e_q:.2e}"
    assert e_k <= t["grad"], f"dk rel-L2 {e_k:.2e}"
    assert e_v <= t["grad"], f"dv rel-L2 {e_v:.2e}"
    return dq, dk, dv


def full_case(cfg, *, backward=True):
    h = inputs.dense_inputs(cfg)
    dev = device_inputs(h)
    out, lse, o_ref, l_ref = check_forward(cfg, h, dev, cfg.splits(), P=cfg.prefix_len,
                                           q_pos0=cfg.q_pos0)
    if backward:
        check_backward(cfg, h, dev, out, lse, o_ref, l_ref, cfg.shard_ranges(),
                       P=cfg.prefix_len, q_pos0=cfg.q_pos0)


# ------------------------------------------------------------------ page gather
@pytest.mark.parametrize("cfg", [
    configs.C1,
    configs.C3.scaled(name="gather_bf16_perm", prefix_len=65536, resp_len=64),
    configs.C3.scaled(name="gather_bf16_p16", page_size=16, prefix_len=4096, resp_len=64),
], ids=lambda c: c.name)
def test_gather_bit_exact(cfg):
    h = inputs.dense_inputs(cfg, with_dout=False)
    dev = device_inputs(h)
    for b, e in ((0, cfg.kv_len), (37, 1111), (cfg.kv_len - 5, cfg.kv_len)):
        announce(f"gather {cfg.name} [{b},{e})")
        k, v = B.gather_kv(_kv(dev), b, e)
        kr = O.gather(h["k_pool"], h["page_table"], cfg.page_size, np.arange(b, e))
        vr = O.gather(h["v_pool"], h["page_table"], cfg.page_size, np.arange(b, e))
        import torch
        as_bits = (lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)) \
            if cfg.dtype == "bf16" else (lambda t: t.cpu().numpy())
        assert np.array_equal(as_bits(k), kr) and np.array_equal(as_bits(v), vr)


# ------------------------------------------------------------------ full parity
def test_c1_tiny_f32():
    full_case(configs.C1)


F32_CASES = [
    # the matrix-core forward (head_dim = head_dim_v in {64, 128}, group a power of two):
    # 16-position pages, unaligned splits, partial row tiles, planted keys
    configs.C1.scaled(name="f32_mfma_d64_g4", n_q_heads=8, n_kv_heads=2, resp_len=77,
                      prefix_len=1000, page_size=16, n_shards=3, splits_per_shard=2,
                      table="perm", plant_frac=0.01),
    configs.C1.scaled(name="f32_mfma_d128_g1", n_q_heads=3, n_kv_heads=3, head_dim=128,
                      head_dim_v=128, resp_len=130, prefix_len=2085, n_shards=2,
                      splits_per_shard=3, table="perm"),
    configs.C1.scaled(name="f32_mfma_d64_g16", n_q_heads=16, n_kv_heads=1, resp_len=9,
                      prefix_len=300, page_size=32, n_shards=1, table="perm"),
    # the generic kernel: other head dims, and a group of three
    configs.C1.scaled(name="f32_generic_d96_g3", n_q_heads=6, n_kv_heads=2, head_dim=96,
                      head_dim_v=96, resp_len=40, prefix_len=700, page_size=16, n_shards=2,
                      table="perm"),
    configs.C1.scaled(name="f32_generic_d64_dv128", head_dim=64, head_dim_v=128, resp_len=50,
                      prefix_len=520, n_shards=2, table="perm"),
    configs.C1.scaled(name="f32_generic_d64_g3", n_q_heads=3, n_kv_heads=1, resp_len=35,
                      prefix_len=400, n_shards=2, table="perm"),
]


@pytest.mark.parametrize("cfg", F32_CASES, ids=lambda c: c.name)
def test_f32_kernels(cfg):
    """fp32 forward on the matrix cores and on the generic kernel, and the
    generic backward, against the oracle at the fp32 tolerance."""
    full_case(cfg)


BF16_SMALL = configs.C3.scaled(name="bf16_small", prefix_len=8192, resp_len=300, n_shards=2,
                               splits_per_shard=2, plant_frac=0.01)


def test_bf16_small_planted():
    full_case(BF16_SMALL)


def test_bf16_small_planted_unit():
    """The secondary planting reading (each planted key moves 4 along the unit
    direction of its target query, the literal "+4 score-sigma")."""
    full_case(BF16_SMALL.scaled(name="bf16_small_unit", plant_unit=True))


def test_bf16_dkdv_row_chunks_and_key_blocks():
    """Response gradients summed over several row chunks of the dk/dv kernel
    and several key blocks, every key and row compared.  640 tokens x G = 8 =
    5,120 packed rows (chunks of 2,048: two full, one partial) against 640
    response keys (five full blocks of 128); 650 tokens = 5,200 rows (a
    partial last 32-row tile) and a sixth block of 10 keys."""
    for r in (640, 650):
        full_case(configs.C3.scaled(name=f"bf16_dkdv_{r}", prefix_len=1024, resp_len=r, n_shards=1,
                                    splits_per_shard=2))


def test_bf16_page16_unaligned_splits():
    cfg = BF16_SMALL.scaled(name="bf16_p16", page_size=16, prefix_len=3000, resp_len=77,
                            plant_frac=0.0)
    h = inputs.dense_inputs(cfg)
    dev = device_inputs(h)
    P = cfg.prefix_len
    splits = [(0, 1000), (1000, 1003), (1003, 2999), (2999, P), (P, P + 40), (P + 40, P + 77)]
    out, lse, o_ref, l_ref = check_forward(cfg, h, dev, splits, P=P, q_pos0=P)
    check_backward(cfg, h, dev, out, lse, o_ref, l_ref, [(0, 1234), (1234, P + 50), (P + 50, P + 77)],
                   P=P, q_pos0=P)


@pytest.mark.parametrize("G,Hkv", [(1, 2), (2, 3), (4, 1), (16, 1), (32, 1)])
def test_bf16_gqa_groups(G, Hkv):
    cfg = BF16_SMALL.scaled(name=f"bf16_g{G}", n_q_heads=G * Hkv, n_kv_heads=Hkv,
                            prefix_len=2048, resp_len=45, plant_frac=0.0, n_shards=1,
                            splits_per_shard=2)
    full_case(cfg)


def test_bf16_few_rows_four_wave_path():
    """At most 128 packed rows take the 4-wave forward on the page path (15
    tokens x G = 8 = 120 rows: one ragged row tile), over several splits."""
    cfg = BF16_SMALL.scaled(name="bf16_r15", prefix_len=6144, resp_len=15, plant_frac=0.0,
                            n_shards=3, splits_per_shard=2)
    full_case(cfg)


@pytest.mark.parametrize("R", [40, 15], ids=["eight_wave", "four_wave"])
def test_bf16_tile_counts(R):
    """Splits and backward ranges of 1 to 6, 15 and 18 key tiles (aligned and ragged), on
    both forward paths (R x G = 8 packed rows: 320 take the two-waves-per-SIMD
    kernel, 120 the pipelined one).  The dense kernels finish the last MFMAs of
    a tile's PV or dq product at the start of the next step, so the one-tile,
    odd and even step counts each take a different way through the loops and
    their tails."""
    P = 1024
    cfg = BF16_SMALL.scaled(name=f"bf16_tiles_r{R}", prefix_len=P, resp_len=R, plant_frac=0.0)
    h = inputs.dense_inputs(cfg)
    dev = device_inputs(h)
    # tiles are the 32-key blocks a range touches
    splits = [(0, 32), (32, 96), (96, 192), (192, 320), (320, 333), (333, 400), (400, 560),
              (560, P), (P, P + R)]
    out, lse, o_ref, l_ref = check_forward(cfg, h, dev, splits, P=P, q_pos0=P)
    ranges = [(0, 32), (32, 96), (96, 200), (200, 331), (331, 480), (480, P + 7), (P + 7, P + R)]
    check_backward(cfg, h, dev, out, lse, o_ref, l_ref, ranges, P=P, q_pos0=P)


def test_bf16_single_row_and_response_only():
    cfg = BF16_SMALL.scaled(name="bf16_r1", prefix_len=512, resp_len=1, plant_frac=0.0,
                            n_shards=1, splits_per_shard=1)
    full_case(cfg)
    cfg = BF16_SMALL.scaled(name="bf16_noprefix", prefix_len=0, resp_len=200, plant_frac=0.0,
                            n_shards=1, splits_per_shard=1)
    h = inputs.dense_inputs(cfg)
    dev = device_inputs(h)
    out, lse, o_ref, l_ref = check_forward(cfg, h, dev, [(0, 200)], P=0, q_pos0=0)
    check_backward(cfg, h, dev, out, lse, o_ref, l_ref, [(0, 200)], P=0, q_pos0=0)


def test_bf16_empty_rows_in_split():
    """A split inside the response: rows before it see nothing (lse -inf, o 0)."""
    cfg = BF16_SMALL.scaled(name="bf16_empty", prefix_len=1024, resp_len=160, plant_frac=0.0)
    h = inputs.dense_inputs(cfg)
    dev = device_inputs(h)
    P = cfg.prefix_len
    announce("fwd empty-row split")
    o_part, l_part = B.prefix_attn_fwd(dev["q"], _kv(dev), [(P + 100, P + 130)], prefix_len=P,
                                       q_pos0=P, scale=cfg.scale)
    o_ref, l_ref = O.attn_fwd(h["q"], h["k_pool"], h["v_pool"], h["page_table"],
                              kv_begin=P + 100, kv_end=P + 130, **oracle_kw(cfg))
    lp = host(l_part[0])
    assert np.all(np.isneginf(lp[:, :100])) and np.all(host(o_part[0])[:100] == 0)
    assert rel_l2(host(o_part[0]), o_ref) <= 5e-3 and lse_err(lp, l_ref) <= 1e-3


def test_bf16_blockwise_q_pos0():
    """Rows start after earlier response keys (a later response block): those keys are
    visible to every row and get dK/dV; accumulating over blocks in reverse equals one
    call over all rows."""
    P, blk, nb = 2048, 96, 3
    cfg = BF16_SMALL.scaled(name="bf16_blocks", prefix_len=P, resp_len=blk * nb, plant_frac=0.0)
    h = inputs.dense_inputs(cfg)
    dev = device_inputs(h)
    import torch
    kv = _kv(dev)
    dk = torch.zeros((blk * nb, cfg.n_kv_heads, 256), dtype=torch.float32, device="cuda")
    dv = torch.zeros_like(dk)
    dq_all = np.zeros((blk * nb, cfg.n_q_heads, 256))
    for b in reversed(range(nb)):
        q0 = P + blk * b
        rows = slice(blk * b, blk * (b + 1))
        q = dev["q"][rows].contiguous()
        d_out = dev["d_out"][rows].contiguous()
        splits = [(0, P), (P, q0 + blk)] if b else [(0, P), (P, P + blk)]
        announce(f"block {b} fwd")
        o_part, l_part = B.prefix_attn_fwd(q, kv, splits, prefix_len=P, q_pos0=q0, scale=cfg.scale)
        out, lse = B.lse_merge(o_part, l_part, out_dtype=torch.bfloat16)
        announce(f"block {b} bwd")
        dq, _, _ = B.prefix_attn_bwd(q, kv, d_out, out, lse, prefix_len=P, q_pos0=q0,
                                     scale=cfg.scale, flags=B.FLAG_ACCUMULATE_DKV,
                                     dk_resp=dk[: q0 + blk - P], dv_resp=dv[: q0 + blk - P])
        torch.cuda.synchronize()
        dq_all[rows] = host(dq)
    dq_ref, dk_ref, dv_ref = O.attn_bwd(h["q"], h["k_pool"], h["v_pool"], h["page_table"],
                                        h["d_out"], **oracle_bkw(cfg))
    assert rel_l2(dq_all, dq_ref) <= 1e-2
    assert rel_l2(host(dk), dk_ref) <= 1e-2
    assert rel_l2(host(dv), dv_ref) <= 1e-2


def test_prep_ready_matches_fresh_prep():
    """ReplayStep runs the prep (Delta, lse * log2(e)) once per backward and
    passes LS_FLAG_PREP_READY for the later key ranges; the gradients are
    bitwise those of calls that each compute their own prep."""
    import torch
    cfg = BF16_SMALL.scaled(name="bf16_prep", n_shards=3)
    dev = device_inputs(inputs.dense_inputs(cfg))
    step = ReplayStep(cfg, dev, backward=True)
    announce("prep reuse: step")
    step.step()
    kv = _kv(dev)
    dq = dk = dv = None
    announce("prep reuse: fresh prep per range")
    for r, (b, e) in enumerate(step.shards):
        dq, dk, dv = B.prefix_attn_bwd(dev["q"], kv, dev["d_out"], step.out, step.lse,
                                       prefix_len=cfg.prefix_len, q_pos0=cfg.q_pos0,
                                       scale=cfg.scale, kv_begin=b, kv_end=e,
                                       flags=B.FLAG_ACCUMULATE_DQ if r else 0, dq=dq, dk_resp=dk,
                                       dv_resp=dv)
    torch.cuda.synchronize()
    assert len(step.shards) == 4
    assert torch.equal(dq, step.dq) and torch.equal(dk, step.dk) and torch.equal(dv, step.dv)


# ------------------------------------------------------------------ invariants
def test_determinism_layout_and_causality():
    cfg = BF16_SMALL.scaled(name="bf16_inv", prefix_len=4096, resp_len=130)
    h = inputs.dense_inputs(cfg)
    dev = device_inputs(h)
    import torch

    def run(d):
        step = ReplayStep(cfg, d)
        step.step()
        torch.cuda.synchronize()
        return [x.clone() for x in (step.out, step.lse, step.dq, step.dk, step.dv)]

    announce("determinism")
    a, b = run(dev), run(dev)
    for x, y in zip(a, b):
        assert torch.equal(x, y), "two runs differ"
    # the same logical store under another physical layout gives identical bits
    perm = np.random.default_rng(0).permutation(h["k_pool"].shape[0])
    inv = np.argsort(perm)
    h2 = dict(h, k_pool=h["k_pool"][perm], v_pool=h["v_pool"][perm],
              page_table=inv[h["page_table"]].astype(np.int32))
    announce("layout invariance")
    c = run(device_inputs(h2))
    for x, y in zip(a, c):
        assert torch.equal(x, y), "physical layout changed the result"
    # changing response token k's K/V leaves rows < k bitwise unchanged
    k = 70
    h3 = dict(h, k_pool=h["k_pool"].copy(), v_pool=h["v_pool"].copy())
    j = cfg.prefix_len + k
    page, slot = h["page_table"][j // cfg.page_size], j % cfg.page_size
    h3["k_pool"][page, slot] ^= np.uint16(0x0100)
    h3["v_pool"][page, slot] ^= np.uint16(0x0100)
    announce("causality")
    d = run(device_inputs(h3))
    assert torch.equal(a[0][:k], d[0][:k]) and torch.equal(a[1][:, :k], d[1][:, :k])
    assert not torch.equal(a[0][k:], d[0][k:])


def test_checked_mode_rejects_bad_page():
    cfg = BF16_SMALL.scaled(name="bf16_oob", prefix_len=1024, resp_len=32, plant_frac=0.0)
    h = inputs.dense_inputs(cfg)
    h["page_table"] = h["page_table"].copy()
    h["page_table"][2] = cfg.n_phys_pages + 5
    dev = device_inputs(h)
    announce("checked mode")
    with pytest.raises(B.LongStrawError) as ei:
        B.prefix_attn_fwd(dev["q"], _kv(dev), [(0, cfg.kv_len)], prefix_len=cfg.prefix_len,
                          q_pos0=cfg.q_pos0, scale=cfg.scale, flags=B.FLAG_CHECKED)
    assert ei.value.name == "LS_ERR_PAGE_OOB"
    with pytest.raises(B.LongStrawError) as ei:
        B.prefix_attn_fwd(dev["q"], _kv(dev, epoch=1), [(0, cfg.kv_len)], prefix_len=cfg.prefix_len,
                          q_pos0=cfg.q_pos0, scale=cfg.scale, expected_epoch=0)
    assert ei.value.name == "LS_ERR_STALE"


# ------------------------------------------------------------------ full-size, sampled
def _sampled_parity(cfg, rows, backward, keys=(), dq_rows=None):
    """The step as bench.py times it, against the oracle on sampled rows (and,
    with backward, the dq of ``dq_rows`` (default: ``rows``) and the dK/dV of
    the response keys ``keys`` (offsets from prefix_len) and the last two, which
    need every row that sees them; those rows' out and lse are compared too).
    The oracle runs over key ranges in a thread pool (tests/_par.py)."""
    h = inputs.dense_inputs(cfg, with_dout=backward)
    if cfg.plant_frac:
        targets = {int(r) for r in h["planted"][1][:2]}
        rows = sorted(set(rows) | targets)
        if dq_rows is not None:
            dq_rows = sorted(set(dq_rows) | targets)
    dev = device_inputs(h)
    announce(f"{cfg.name} full step")
    step = ReplayStep(cfg, dev, backward=backward)
    step.step()
    import torch
    torch.cuda.synchronize()
    R = cfg.resp_len
    rows = np.unique(np.asarray(rows))
    dq_rows = rows if dq_rows is None else np.unique(np.asarray(dq_rows))
    keys = np.unique(np.concatenate([np.asarray(keys, np.int64), [R - 2, R - 1]])) + cfg.prefix_len
    need = np.union1d(rows, np.arange(int(keys.min()) - cfg.prefix_len, R)) if backward else rows
    need = np.union1d(need, dq_rows) if backward else need
    kw = dict(oracle_kw(cfg), prefix_len=cfg.prefix_len)
    o_n, l_n = _par.dense_fwd(h, rows=need, **kw)
    assert rel_l2(host(step.out)[need], o_n) <= 5e-3, "out"
    assert lse_err(host(step.lse)[:, need], l_n) <= 1e-3, "lse"
    if backward:
        o_full = np.zeros((R, cfg.n_q_heads, cfg.head_dim_v))
        l_full = np.zeros((cfg.n_q_heads, R))
        o_full[need], l_full[:, need] = o_n, l_n
        dq_ref, dk_ref, dv_ref = _par.dense_bwd(h, rows=dq_rows, resp_keys=keys, out=o_full,
                                                lse=l_full, **kw)
        assert rel_l2(host(step.dq)[dq_rows], dq_ref) <= 1e-2, "dq"
        # every response key on its own (a bad key would be diluted in one norm)
        k_off = keys - cfg.prefix_len
        for name, got, ref in (("dk", host(step.dk)[k_off], dk_ref), ("dv", host(step.dv)[k_off], dv_ref)):
            err = np.linalg.norm((got - ref).reshape(len(k_off), -1), axis=1)
            err /= np.linalg.norm(ref.reshape(len(k_off), -1), axis=1)
            worst = int(np.argmax(err))
            assert err[worst] <= 1e-2, f"{name} of response key {k_off[worst]}: rel-L2 {err[worst]:.2e}"


def _wg_boundary_rows(n_tokens, tokens_per_wg, every=1, inner=()):
    """First and last token of every `every`-th workgroup (plus `inner` offsets)."""
    out = []
    for b in range(0, n_tokens, tokens_per_wg * every):
        out += [b, b + tokens_per_wg - 1] + [b + o for o in inner]
    return [r for r in out if r < n_tokens]


@pytest.mark.timeout(900)
def test_c2_full_size():
    """c2 as bench.py's forward-only configuration runs it: every one of the
    4,096 tokens' out and lse (16 heads over 262,144 prefix keys), against the
    fp64 oracle composed over key ranges."""
    _sampled_parity(configs.C2, np.arange(configs.C2.resp_len), backward=False)


@pytest.mark.timeout(1200)
def test_c3_full_size():
    """c3 as bench.py times it: every row's out and lse (4,096 tokens x 16
    heads over 2,101,248 keys) and every response key's dK/dV (each through
    the ordered reduction over the dK/dV row chunks that see it), and dq on
    513+ rows: both sides of the dq (16-token) and forward (32-token)
    workgroup boundaries in every forward workgroup, the last row, and planted
    targets."""
    R = configs.C3.resp_len
    dq_rows = _wg_boundary_rows(R, 32, every=1, inner=(15, 16)) + [R - 1]
    _sampled_parity(configs.C3, np.arange(R), backward=True, keys=np.arange(R), dq_rows=dq_rows)


@pytest.mark.timeout(900)
def test_c3_cyclic_bf16_numerator_full_size_sampled():
    """c3 as the paper's production composition runs it: pages dealt to 8
    shards by owner(p) = p mod 8 and the cross-shard numerator reduced in
    bf16; sampled rows and response keys against the unsharded fp64 oracle."""
    _sampled_parity(configs.C3.scaled(ownership="cyclic", bf16_numerator=True), [1, 3000, 4094],
                    backward=True)


def test_response_full_chunk_reduction():
    """The c3 response geometry (4,096 tokens, 16 query heads on 2 KV heads: 16
    dK/dV row chunks x 32 key blocks x 2 heads) over a 2,048-position prefix:
    every response key's dK/dV, and every row's out, lse and dq, in full."""
    cfg = configs.C3.scaled(name="c3_resp_geometry", prefix_len=2048, n_shards=1,
                            splits_per_shard=1, plant_frac=0.0)
    h = inputs.dense_inputs(cfg)
    dev = device_inputs(h)
    announce(cfg.name)
    step = ReplayStep(cfg, dev, backward=True)
    step.step()
    import torch
    torch.cuda.synchronize()
    R = cfg.resp_len
    rows = np.arange(R)
    kw = dict(oracle_kw(cfg), prefix_len=cfg.prefix_len)
    o_n, l_n = _par.dense_fwd(h, rows=rows, piece=1024, **kw)
    assert rel_l2(host(step.out), o_n) <= 5e-3
    assert lse_err(host(step.lse), l_n) <= 1e-3
    keys = cfg.prefix_len + np.arange(R)
    dq_ref, dk_ref, dv_ref = _par.dense_bwd(h, rows=rows, resp_keys=keys, out=o_n, lse=l_n,
                                            piece=1024, **kw)
    assert rel_l2(host(step.dq), dq_ref) <= 1e-2
    assert rel_l2(host(step.dk), dk_ref) <= 1e-2
    assert rel_l2(host(step.dv), dv_ref) <= 1e-2
