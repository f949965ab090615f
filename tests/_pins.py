"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each pin takes the oracle module ``O`` and raises AssertionError when the
module disagrees with a closed form, an invariant, a library routine or brute
force.  ``test_oracle_pins.py`` runs them on the real oracle;
``test_oracle_mutations.py`` runs them on copies of the oracle with planted
mistakes and requires that every mistake trips at least one pin.
"""
from __future__ import annotations

import numpy as np

from tests._tiny import make, rel_l2


def _close(a, b, tol, what):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    fin = np.isfinite(b)
    assert np.array_equal(np.isfinite(a), fin), f"{what}: finiteness differs"
    err = np.max(np.abs(a[fin] - b[fin]) / (1.0 + np.abs(b[fin]))) if fin.any() else 0.0
    assert err <= tol, f"{what}: err {err:.3e} > {tol:.1e}"


# ---------------------------------------------------------------- forward closed forms
def pin_single_key(O):
    """A range holding one visible key gives o = v_j and lse = s_ij
    (Eq. qwen-local-attn with |K_r| = 1)."""
    t = make(P=40, R=5, Hq=4, Hkv=2, D=8, S=8, seed=1)
    G = 2
    for j in (0, 17, 39):
        o, lse = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, kv_begin=j, kv_end=j + 1, **t.kw())
        for h in range(4):
            g = h // G
            page, slot = t.page_table[j // t.S], j % t.S
            k, v = t.k_pool[page, slot, g], t.v_pool[page, slot, g]
            _close(o[:, h], np.broadcast_to(v, o[:, h].shape), 1e-13, "single key o")
            _close(lse[h], t.scale * (t.q[:, h] @ k), 1e-13, "single key lse")
    # response key P + i is first visible to row i: row i sees exactly one key of [P+i, P+i+1)
    for i in range(t.R):
        o, lse = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table,
                            kv_begin=t.P + i, kv_end=t.P + i + 1, **t.kw())
        assert np.all(np.isneginf(lse[:, :i])) and np.all(o[:i] == 0), "rows before i see key P+i"
        assert np.all(np.isfinite(lse[:, i:])), "rows from i on must see key P+i"


def pin_identical_keys(O):
    """All keys equal: o is the mean of the visible values and
    lse = s + ln|V_i| with |V_i| = q_pos0 + i + 1 (inclusive causal count)."""
    t = make(P=33, R=7, Hq=6, Hkv=2, D=8, S=8, seed=2)
    rng = np.random.default_rng(7)
    kk = rng.standard_normal((2, 8))
    for g in range(2):
        t.set_rows("k_pool", np.arange(t.kv_len), g, kk[g])
    o, lse = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, **t.kw())
    for h in range(6):
        g = h // 3
        V = np.stack([t.v_pool[t.page_table[j // t.S], j % t.S, g] for j in range(t.kv_len)])
        for i in range(t.R):
            n = t.P + i + 1
            _close(o[i, h], V[:n].mean(axis=0), 1e-12, "identical keys mean")
            _close(lse[h, i], t.scale * (t.q[i, h] @ kk[g]) + np.log(n), 1e-12, "identical keys lse")


def pin_zero_query(O):
    """q = 0 gives the uniform mean and lse = ln|V_i| over any range."""
    t = make(P=50, R=6, Hq=2, Hkv=1, D=4, S=16, seed=3)
    t.q[:] = 0.0
    b, e = 10, 53
    o, lse = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, kv_begin=b, kv_end=e, **t.kw())
    V = np.stack([t.v_pool[t.page_table[j // t.S], j % t.S, 0] for j in range(t.kv_len)])
    for i in range(t.R):
        hi = min(e, t.P + i + 1)
        _close(lse[:, i], np.full(2, np.log(hi - b)), 1e-13, "zero query lse")
        _close(o[i], np.broadcast_to(V[b:hi].mean(axis=0), (2, 4)), 1e-12, "zero query o")


def pin_scale_and_gqa(O):
    """Two keys with known scores: o = sigmoid-weighted mix, lse = log(e^s1 + e^s2),
    and head h reads KV head h // (Hq/Hkv)."""
    t = make(P=2, R=1, Hq=4, Hkv=2, D=4, S=2, seed=4, table="identity", extra_pages=0, scale=0.5)
    o, lse = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, kv_begin=0, kv_end=2, **t.kw())
    for h in range(4):
        g = h // 2
        k0, k1 = t.k_pool[0, 0, g], t.k_pool[0, 1, g]
        v0, v1 = t.v_pool[0, 0, g], t.v_pool[0, 1, g]
        s0, s1 = 0.5 * t.q[0, h] @ k0, 0.5 * t.q[0, h] @ k1
        w1 = 1.0 / (1.0 + np.exp(s0 - s1))
        _close(o[0, h], (1 - w1) * v0 + w1 * v1, 1e-13, "two-key mix")
        _close(lse[h, 0], np.logaddexp(s0, s1), 1e-13, "two-key lse")


# ---------------------------------------------------------------- merge
def pin_merge_closed_form(O):
    """Parts with l1 = ln 2, l2 = ln 3 compose to (2 o1 + 3 o2) / 5 and ln 5
    (Eq. qwen-lse-parts, Eq. qwen-global-attn); an empty part (-inf) has weight 0."""
    o1 = np.full((1, 1, 3), 1.0)
    o2 = np.array([[[2.0, -1.0, 4.0]]])
    oe = np.zeros((1, 1, 3))
    l1, l2, le = np.log([[2.0]]), np.log([[3.0]]), np.array([[-np.inf]])
    o, lse = O.lse_merge([o1, oe, o2], [l1, le, l2])
    _close(o, (2 * o1 + 3 * o2) / 5, 1e-14, "merge o")
    _close(lse, np.log([[5.0]]), 1e-14, "merge lse")
    # large offsets stay finite (the max shift)
    o, lse = O.lse_merge([o1, o2], [l1 + 900.0, l2 + 900.0])
    _close(lse, np.log([[5.0]]) + 900.0, 1e-14, "merge shift")
    # all parts empty -> o = 0, lse = -inf
    o, lse = O.lse_merge([oe, oe], [le, le])
    assert np.all(o == 0) and np.all(np.isneginf(lse)), "all-empty merge"


def pin_split_merge_invariance(O):
    """Any partition of the keys, each range computed alone and merged, equals the
    unsplit result; merging one part is the identity; order does not matter."""
    t = make(P=70, R=9, Hq=4, Hkv=1, D=8, S=8, seed=5)
    full_o, full_l = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, **t.kw())
    rng = np.random.default_rng(11)
    for trial in range(6):
        cuts = np.sort(rng.choice(np.arange(1, t.kv_len), size=rng.integers(1, 6), replace=False))
        bounds = [0, *cuts.tolist(), t.kv_len]
        parts = [O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, kv_begin=b, kv_end=e, **t.kw())
                 for b, e in zip(bounds[:-1], bounds[1:])]
        order = rng.permutation(len(parts))
        o, l = O.lse_merge([parts[k][0] for k in order], [parts[k][1] for k in order])
        _close(o, full_o, 1e-12, "split+merge o")
        _close(l, full_l, 1e-12, "split+merge lse")
    o, l = O.lse_merge([full_o], [full_l])
    _close(o, full_o, 1e-15, "merge identity o")
    _close(l, full_l, 1e-15, "merge identity lse")


def pin_causal(O):
    """Changing response token k's K/V leaves rows i < k exactly unchanged and
    changes every row i >= k."""
    t = make(P=24, R=8, Hq=2, Hkv=1, D=4, S=8, seed=6)
    o0, l0 = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, **t.kw())
    k = 3
    t.set_rows("k_pool", [t.P + k], 0, 3.0)
    t.set_rows("v_pool", [t.P + k], 0, -5.0)
    o1, l1 = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, **t.kw())
    assert np.array_equal(o0[:k], o1[:k]) and np.array_equal(l0[:, :k], l1[:, :k]), "earlier rows moved"
    assert np.all(np.abs(o0[k:] - o1[k:]).max(axis=(1, 2)) > 1e-6), "later rows unchanged"


# ---------------------------------------------------------------- paged store
def pin_gather_bruteforce(O):
    """The paged gather equals a scalar loop over (page, slot), bit for bit, and a
    permuted pool with the matching table gives the same attention bit for bit."""
    t = make(P=37, R=5, Hq=2, Hkv=2, D=3, S=4, seed=8, dtype=np.float32)
    pos = np.arange(5, t.kv_len)
    got = O.gather(t.k_pool, t.page_table, t.S, pos)
    for n, j in enumerate(pos):
        page = int(t.page_table[j // t.S])
        for g in range(2):
            for d in range(3):
                assert got[n, g, d] == t.k_pool[page, j % t.S, g, d], "gather"
    perm = np.random.default_rng(3).permutation(t.k_pool.shape[0])
    inv = np.argsort(perm)
    k2, v2 = t.k_pool[perm], t.v_pool[perm]        # physical page p moves to inv[p]
    pt2 = inv[t.page_table].astype(np.int32)
    a = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, **t.kw())
    b = O.attn_fwd(t.q, k2, v2, pt2, **t.kw())
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]), "layout changed the result"


# ---------------------------------------------------------------- backward
def _loss(O, t):
    o, _ = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, **t.kw())
    return float(np.sum(t.d_out * o))


def pin_finite_differences(O):
    """dq, dk_resp, dv_resp equal central differences of L = sum(dO * O); prefix K/V
    are stop-gradient state and have no entry (Eq. gradient-boundary)."""
    t = make(P=20, R=6, Hq=2, Hkv=1, D=4, S=8, seed=9)
    dq, dk, dv = O.attn_bwd(t.q, t.k_pool, t.v_pool, t.page_table, t.d_out, **t.bkw())
    assert dk.shape == (t.R, 1, 4) and dv.shape == (t.R, 1, 4), "response-only dk/dv"
    h = 1e-6
    num = np.zeros_like(t.q)
    for idx in np.ndindex(t.q.shape):
        base = t.q[idx]
        t.q[idx] = base + h; lp = _loss(O, t)
        t.q[idx] = base - h; lm = _loss(O, t)
        t.q[idx] = base
        num[idx] = (lp - lm) / (2 * h)
    assert rel_l2(dq, num) < 1e-6, f"dq vs finite differences {rel_l2(dq, num):.2e}"
    for name, grad in (("k_pool", dk), ("v_pool", dv)):
        pool = getattr(t, name)
        num = np.zeros_like(grad)
        for i in range(t.R):
            j = t.P + i
            page, slot = t.page_table[j // t.S], j % t.S
            for d in range(pool.shape[3]):
                base = pool[page, slot, 0, d]
                pool[page, slot, 0, d] = base + h; lp = _loss(O, t)
                pool[page, slot, 0, d] = base - h; lm = _loss(O, t)
                pool[page, slot, 0, d] = base
                num[i, 0, d] = (lp - lm) / (2 * h)
        assert rel_l2(grad, num) < 1e-6, f"{name} vs finite differences {rel_l2(grad, num):.2e}"


def pin_bwd_partition(O):
    """dq over a partition of the keys sums to the full dq (Eq. qwen-dq-reduce);
    dk/dv of a range are the matching rows of the full response gradient."""
    t = make(P=40, R=10, Hq=4, Hkv=2, D=4, S=8, seed=10)
    dq, dk, dv = O.attn_bwd(t.q, t.k_pool, t.v_pool, t.page_table, t.d_out, **t.bkw())
    acc = np.zeros_like(dq)
    for b, e in ((0, 13), (13, 40), (40, 44), (44, 50)):
        dq_r, dk_r, dv_r = O.attn_bwd(t.q, t.k_pool, t.v_pool, t.page_table, t.d_out,
                                      kv_begin=b, kv_end=e, **t.bkw())
        acc += dq_r
        lo, hi = max(b, t.P) - t.P, max(e, t.P) - t.P
        _close(dk_r, dk[lo:hi], 1e-12, "range dk")
        _close(dv_r, dv[lo:hi], 1e-12, "range dv")
    _close(acc, dq, 1e-12, "dq partition sum")


def _torch_dense(t):
    """Dense masked softmax attention in torch fp64 with autograd; the prefix K/V
    are detached leaves, the response K/V carry gradient."""
    import torch
    R, Hq, D = t.q.shape
    Hkv = t.k_pool.shape[2]
    G = Hq // Hkv
    n = t.kv_len
    K = np.zeros((n, Hkv, D)); V = np.zeros((n, Hkv, t.v_pool.shape[3]))
    for j in range(n):                                   # brute-force page walk
        page, slot = int(t.page_table[j // t.S]), j % t.S
        K[j], V[j] = t.k_pool[page, slot], t.v_pool[page, slot]
    q = torch.tensor(t.q, dtype=torch.float64, requires_grad=True)
    k_pre = torch.tensor(K[:t.P])
    v_pre = torch.tensor(V[:t.P])
    k_resp = torch.tensor(K[t.P:], requires_grad=True)
    v_resp = torch.tensor(V[t.P:], requires_grad=True)
    Kt = torch.cat([k_pre, k_resp])
    Vt = torch.cat([v_pre, v_resp])
    mask = torch.arange(n)[None, :] > (t.P + torch.arange(R))[:, None]
    outs, lses = [], []
    for h in range(Hq):
        g = h // G
        s = t.scale * q[:, h] @ Kt[:, g].T
        s = s.masked_fill(mask, float("-inf"))
        lses.append(torch.logsumexp(s, dim=1))
        outs.append(torch.softmax(s, dim=1) @ Vt[:, g])
    out = torch.stack(outs, dim=1)
    lse = torch.stack(lses)
    (out * torch.tensor(t.d_out)).sum().backward()
    return (out.detach().numpy(), lse.detach().numpy(), q.grad.numpy(),
            k_resp.grad.numpy(), v_resp.grad.numpy())


def pin_torch_autograd(O):
    """Forward and response-only backward equal torch's softmax/logsumexp with
    autograd on a dense masked problem (an independent code path)."""
    t = make(P=45, R=11, Hq=6, Hkv=2, D=8, Dv=5, S=8, seed=12)
    out, lse, dq_t, dk_t, dv_t = _torch_dense(t)
    o, l = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, **t.kw())
    _close(o, out, 1e-12, "torch o")
    _close(l, lse, 1e-12, "torch lse")
    dq, dk, dv = O.attn_bwd(t.q, t.k_pool, t.v_pool, t.page_table, t.d_out, **t.bkw())
    _close(dq, dq_t, 1e-11, "torch dq")
    _close(dk, dk_t, 1e-11, "torch dk")
    _close(dv, dv_t, 1e-11, "torch dv")


def pin_sampled_rows(O):
    """Row/key subsets used at large sizes equal slices of the full result."""
    t = make(P=64, R=12, Hq=4, Hkv=2, D=4, S=8, seed=13)
    o, l = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, **t.kw())
    rows = np.array([0, 5, 11])
    o2, l2 = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, rows=rows, heads=[1, 3], **t.kw())
    _close(o2, o[rows][:, [1, 3]], 1e-14, "row subset o")
    _close(l2, l[[1, 3]][:, rows], 1e-14, "row subset lse")
    dq, dk, dv = O.attn_bwd(t.q, t.k_pool, t.v_pool, t.page_table, t.d_out, **t.bkw())
    keys = np.array([t.P + 9, t.P + 11])
    dq2, dk2, dv2 = O.attn_bwd(t.q, t.k_pool, t.v_pool, t.page_table, t.d_out, rows=rows,
                               resp_keys=keys, **t.bkw())
    _close(dq2, dq[rows], 1e-12, "row subset dq")
    _close(dk2, dk[[9, 11]], 1e-12, "key subset dk")
    _close(dv2, dv[[9, 11]], 1e-12, "key subset dv")
    # one KV head: its group's query heads in dq, its own dK/dV, all unchanged
    dq3, dk3, dv3 = O.attn_bwd(t.q, t.k_pool, t.v_pool, t.page_table, t.d_out, rows=rows,
                               resp_keys=keys, kv_heads=[1], **t.bkw())
    _close(dq3, dq[rows][:, [2, 3]], 1e-12, "KV head subset dq")
    _close(dk3, dk[[9, 11]][:, [1]], 1e-12, "KV head subset dk")
    _close(dv3, dv[[9, 11]][:, [1]], 1e-12, "KV head subset dv")


# ---------------------------------------------------------------- sparse latent replay
def _latent(P=30, R=5, H=3, Dk=6, Dv=4, S=4, seed=14):
    t = make(P=P, R=R, Hq=H, Hkv=1, D=Dk, Dv=Dk, S=S, seed=seed)
    t.v_pool = t.k_pool                                    # values alias the latent rows
    return t, Dv


def pin_sparse_full_index_is_dense(O):
    """With every prefix position selected, sparse latent replay equals dense
    attention with keys = the latent row and values = its first Dv channels."""
    t, Dv = _latent()
    idx = np.tile(np.arange(t.P, dtype=np.int32), (t.R, 1))
    so, sl = O.sparse_fwd(t.q, t.k_pool, t.page_table, idx, page_size=t.S, prefix_len=t.P,
                          q_pos0=t.P, scale=t.scale, head_dim_v=Dv)
    do, dl = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, head_dim_v=Dv, **t.kw())
    _close(so, do, 1e-12, "sparse=dense o")
    _close(sl, dl, 1e-12, "sparse=dense lse")
    d_out = t.d_out[..., :Dv]
    sdq = O.sparse_bwd(t.q, t.k_pool, t.page_table, idx, d_out, page_size=t.S, prefix_len=t.P,
                       q_pos0=t.P, scale=t.scale, head_dim_v=Dv)
    ddq, _, _ = O.attn_bwd(t.q, t.k_pool, t.v_pool, t.page_table, d_out, head_dim_v=Dv, **t.bkw())
    _close(sdq, ddq, 1e-11, "sparse=dense dq")


def pin_sparse_subset(O):
    """A sparse selection equals dense attention over exactly the selected keys
    (brute force per row), and dq matches central differences."""
    t, Dv = _latent(P=24, R=4, seed=15)
    rng = np.random.default_rng(5)
    idx = np.stack([np.sort(rng.choice(t.P, 7, replace=False)) for _ in range(t.R)]).astype(np.int32)
    so, sl = O.sparse_fwd(t.q, t.k_pool, t.page_table, idx, page_size=t.S, prefix_len=t.P,
                          q_pos0=t.P, scale=t.scale, head_dim_v=Dv)
    for i in range(t.R):
        keys = list(idx[i]) + list(range(t.P, t.P + i + 1))
        C = np.stack([t.k_pool[t.page_table[j // t.S], j % t.S, 0] for j in keys])
        for h in range(t.q.shape[1]):
            s = t.scale * C @ t.q[i, h]
            w = np.exp(s - s.max())
            _close(so[i, h], (w / w.sum()) @ C[:, :Dv], 1e-12, "sparse brute o")
            _close(sl[h, i], s.max() + np.log(w.sum()), 1e-12, "sparse brute lse")
    d_out = t.d_out[..., :Dv]
    dq = O.sparse_bwd(t.q, t.k_pool, t.page_table, idx, d_out, page_size=t.S, prefix_len=t.P,
                      q_pos0=t.P, scale=t.scale, head_dim_v=Dv)
    h = 1e-6
    num = np.zeros_like(t.q)
    for ix in np.ndindex(t.q.shape):
        base = t.q[ix]
        vals = []
        for d in (h, -h):
            t.q[ix] = base + d
            o, _ = O.sparse_fwd(t.q, t.k_pool, t.page_table, idx, page_size=t.S, prefix_len=t.P,
                                q_pos0=t.P, scale=t.scale, head_dim_v=Dv)
            vals.append(np.sum(d_out * o))
        t.q[ix] = base
        num[ix] = (vals[0] - vals[1]) / (2 * h)
    assert rel_l2(dq, num) < 1e-6, f"sparse dq vs finite differences {rel_l2(dq, num):.2e}"


def pin_sparse_invalid_entries(O):
    """Selection entries outside the prefix select nothing: a row whose entries
    are all -1 pads sees only its response window (the first row: its own
    latent row, so o = its first Dv channels and lse = s), and a selection with
    pads or out-of-prefix entries equals brute force over its valid entries."""
    t, Dv = _latent(P=20, R=4, seed=16)
    idx = np.array([[-1, -1, -1, -1, -1],
                    [3, -1, 11, -1, -1],
                    [0, 19, 20, 22, -1],      # 20 and 22 are response positions: no key
                    [5, 6, 7, 8, 9]], dtype=np.int32)
    so, sl = O.sparse_fwd(t.q, t.k_pool, t.page_table, idx, page_size=t.S, prefix_len=t.P,
                          q_pos0=t.P, scale=t.scale, head_dim_v=Dv)
    own = t.k_pool[t.page_table[t.P // t.S], t.P % t.S, 0]
    _close(so[0], np.broadcast_to(own[:Dv], so[0].shape), 1e-13, "pads only: o = own value")
    _close(sl[:, 0], t.scale * (t.q[0] @ own), 1e-13, "pads only: lse = own score")
    for i in range(t.R):
        keys = [j for j in idx[i] if 0 <= j < t.P] + list(range(t.P, t.P + i + 1))
        C = np.stack([t.k_pool[t.page_table[j // t.S], j % t.S, 0] for j in keys])
        for h in range(t.q.shape[1]):
            s = t.scale * C @ t.q[i, h]
            w = np.exp(s - s.max())
            _close(so[i, h], (w / w.sum()) @ C[:, :Dv], 1e-12, "sparse pads brute o")
            _close(sl[h, i], s.max() + np.log(w.sum()), 1e-12, "sparse pads brute lse")
    d_out = t.d_out[..., :Dv]
    dq = O.sparse_bwd(t.q, t.k_pool, t.page_table, idx, d_out, page_size=t.S, prefix_len=t.P,
                      q_pos0=t.P, scale=t.scale, head_dim_v=Dv)
    for i in range(t.R):
        keys = [j for j in idx[i] if 0 <= j < t.P] + list(range(t.P, t.P + i + 1))
        C = np.stack([t.k_pool[t.page_table[j // t.S], j % t.S, 0] for j in keys])
        for h in range(t.q.shape[1]):
            s = t.scale * C @ t.q[i, h]
            P_ = np.exp(s - s.max())
            P_ /= P_.sum()
            o = P_ @ C[:, :Dv]
            dS = P_ * (C[:, :Dv] @ d_out[i, h] - d_out[i, h] @ o)
            _close(dq[i, h], t.scale * dS @ C, 1e-12, "sparse pads brute dq")


# ---------------------------------------------------------------- input decoding
def pin_decode(O):
    """bf16 bit patterns decode to the values the bfloat16 format defines
    (sign, 8-bit exponent with bias 127, 7-bit fraction; the upper half of the
    fp32 encoding): hand-made patterns against their exact values, every one of
    the 65,536 patterns against torch's bfloat16 -> float64 cast, and fp32
    input passed through unchanged."""
    import torch
    hand = {
        0x3F80: 1.0, 0xBF80: -1.0, 0xC020: -2.5, 0x4049: 3.140625, 0x4000: 2.0,
        0x3F00: 0.5, 0x3FC0: 1.5, 0x3F81: 1.0 + 2.0 ** -7, 0x0080: 2.0 ** -126,
        0x0001: 2.0 ** -133, 0x007F: 127 * 2.0 ** -133, 0x7F7F: (2.0 - 2.0 ** -7) * 2.0 ** 127,
        0x4780: 65536.0, 0xC7C3: -99840.0,
    }
    bits = np.array(list(hand), dtype=np.uint16)
    got = O.decode(bits)
    assert got.dtype == np.float64, "decode must return float64"
    assert np.array_equal(got, np.array(list(hand.values()))), f"decode of hand patterns: {got}"
    z = O.decode(np.array([0x0000, 0x8000], dtype=np.uint16))
    assert np.array_equal(z, [0.0, 0.0]) and not np.signbit(z[0]) and np.signbit(z[1]), "signed zeros"
    inf = O.decode(np.array([0x7F80, 0xFF80], dtype=np.uint16))
    assert np.array_equal(inf, [np.inf, -np.inf]), "infinities"
    assert np.all(np.isnan(O.decode(np.array([0x7FC0, 0xFFC1, 0x7F81], dtype=np.uint16)))), "NaNs"
    every = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    want = torch.from_numpy(every.view(np.int16).copy()).view(torch.bfloat16).to(torch.float64).numpy()
    got = O.decode(every)
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan), "decode: NaN patterns differ from torch"
    assert np.array_equal(got[~nan], want[~nan]), "decode differs from torch's bfloat16 cast"
    rng = np.random.default_rng(22)
    x = rng.standard_normal((3, 5)).astype(np.float32)
    assert np.array_equal(O.decode(x), x.astype(np.float64)), "fp32 input must pass through"
    shaped = O.decode(every[:24].reshape(2, 3, 4))
    assert shaped.shape == (2, 3, 4) and np.array_equal(shaped.ravel(), O.decode(every[:24])), "shape"


# ---------------------------------------------------------------- production composition
def pin_bf16_round(O):
    """bf16 rounding equals torch's float32 -> bfloat16 cast (round to nearest
    even) on float32 values, and hand-checked ties: 1 + 2^-8 -> 1 (even),
    1 + 3 * 2^-8 -> 1 + 2^-6 (even), -(1 + 2^-7 + 2^-9) -> -(1 + 2^-7)."""
    import torch
    rng = np.random.default_rng(21)
    x = (rng.standard_normal(4096) * np.exp2(rng.integers(-30, 30, 4096))).astype(np.float32)
    x[:8] = [1.0, 0.0, -2.5, 3.0e38, 1.17549435e-38, 65504.0, 1.0 / 3, -7.0]
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = O.bf16_round(x.astype(np.float64))
    assert np.array_equal(got, want), "bf16 rounding differs from torch's cast"
    ties = np.array([1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, -(1 + 2.0 ** -7 + 2.0 ** -9)])
    assert np.array_equal(O.bf16_round(ties), [1.0, 1 + 2.0 ** -6, -(1 + 2.0 ** -7)]), "bf16 ties"


def pin_bf16_numerator_merge(O):
    """The bf16-numerator composition: one part gives bf16(o); terms are
    rounded and the sum is rounded after every addition, in part order
    (1, 2^-8, 2^-8 sums to 1, but 2^-8, 2^-8, 1 to 1 + 2^-7); m, a and l stay
    exact; with bf16-exact terms and sums it equals the exact merge."""
    rng = np.random.default_rng(22)
    o1 = rng.standard_normal((3, 2, 5))
    l1 = rng.standard_normal((2, 3))
    o, lse = O.lse_merge_bf16_numerator([o1], [l1])
    assert np.array_equal(o, O.bf16_round(o1)), "one part: o = bf16(o)"
    _close(lse, l1, 1e-15, "one part: lse")
    ones = np.zeros((1, 1))
    parts = [np.full((1, 1, 1), 1.0), np.full((1, 1, 1), 2.0 ** -8), np.full((1, 1, 1), 2.0 ** -8)]
    o, lse = O.lse_merge_bf16_numerator(parts, [ones, ones, ones])
    assert o[0, 0, 0] == 1.0 / 3, "running sum rounded after each addition"
    _close(lse, np.log([[3.0]]), 1e-15, "lse with the exact denominator")
    o, _ = O.lse_merge_bf16_numerator(parts[::-1], [ones, ones, ones])
    assert o[0, 0, 0] == (1 + 2.0 ** -7) / 3, "parts summed in the given order"
    # bf16-exact data: small integers with weights 1, 1/2 (l = 0, -ln 2)
    oa = rng.integers(-8, 8, (4, 3, 6)).astype(np.float64)
    ob = rng.integers(-8, 8, (4, 3, 6)).astype(np.float64) * 2.0
    la, lb = np.zeros((3, 4)), np.full((3, 4), -np.log(2.0))
    want_o, want_l = O.lse_merge([oa, ob], [la, lb])
    got_o, got_l = O.lse_merge_bf16_numerator([oa, ob], [la, lb])
    _close(got_o, want_o, 1e-15, "bf16-exact merge o")
    _close(got_l, want_l, 1e-15, "bf16-exact merge lse")
    # random data: within the rounding bound of S terms and S - 1 additions
    parts = [rng.standard_normal((6, 2, 8)) for _ in range(5)]
    lses = [rng.standard_normal((2, 6)) for _ in range(5)]
    eo, _ = O.lse_merge(parts, lses)
    go, _ = O.lse_merge_bf16_numerator(parts, lses)
    bound = 10 * 2.0 ** -9 * np.max(np.abs(np.stack(parts)))
    assert np.max(np.abs(go - eo)) <= bound, "bf16 numerator error bound"
    assert np.max(np.abs(go - eo)) > 0, "bf16 numerator must round"


def pin_cyclic_ownership(O):
    """owner(p) = p mod C (Eq. qwen-page-owner): the shards' positions
    partition the prefix, shard c holds exactly the pages congruent to c, and
    composing the shards' results with the response range equals the unsplit
    forward."""
    t = make(P=75, R=6, Hq=4, Hkv=2, D=8, S=8, seed=23)
    C = 3
    owned = [O.cyclic_owned_positions(t.P, t.S, C, c) for c in range(C)]
    allp = np.sort(np.concatenate(owned))
    assert np.array_equal(allp, np.arange(t.P)), "shards partition the prefix"
    for c in range(C):
        assert np.all((owned[c] // t.S) % C == c), "shard c owns pages p with p mod C = c"
        assert np.all(np.diff(owned[c]) > 0), "positions in increasing order"
    full_o, full_l = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, **t.kw())
    parts = [O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, key_positions=owned[c], **t.kw())
             for c in range(C)]
    parts.append(O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, kv_begin=t.P,
                            kv_end=t.kv_len, **t.kw()))
    o, lse = O.lse_merge([p[0] for p in parts], [p[1] for p in parts])
    _close(o, full_o, 1e-12, "cyclic shards o")
    _close(lse, full_l, 1e-12, "cyclic shards lse")
    # a key set given as positions equals the same contiguous range
    a = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, kv_begin=10, kv_end=50, **t.kw())
    b = O.attn_fwd(t.q, t.k_pool, t.v_pool, t.page_table, key_positions=np.arange(10, 50), **t.kw())
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]), "positions == range"


# ---------------------------------------------------------------- DSA index selection
def pin_dsa_index_closed_form(O):
    """Eq. dsa-index on hand-made keys: one head with weight 1 gives ReLU(q.k)
    (negative dot products give 0); weights scale each head's term linearly and
    may be negative; the page layout does not matter."""
    S, d = 4, 3
    k_dense = np.array([[1.0, 0, 0], [0, 1.0, 0], [-1.0, 0, 0], [0, 0, 2.0],
                        [1.0, 1.0, 1.0], [0, -2.0, 0], [0.5, 0, 0], [0, 0, -1.0]])
    pool = k_dense.reshape(2, S, d)
    ident = np.arange(2, dtype=np.int32)
    q = np.array([[[2.0, 3.0, -1.0], [1.0, -1.0, 1.0]]])              # [R=1, H=2, d]
    w1 = np.array([[1.0, 0.0]])
    got = O.dsa_index_scores(q, w1, pool, ident, page_size=S, pos_begin=0, pos_end=8)
    want = np.maximum(k_dense @ q[0, 0], 0.0)[None]
    _close(got, want, 1e-15, "one head, weight 1")
    assert got[0, 2] == 0.0 and got[0, 5] == 0.0, "negative dot products give 0"
    w2 = np.array([[2.0, -0.5]])
    got = O.dsa_index_scores(q, w2, pool, ident, page_size=S, pos_begin=2, pos_end=7)
    want = (2.0 * np.maximum(k_dense @ q[0, 0], 0) - 0.5 * np.maximum(k_dense @ q[0, 1], 0))[2:7]
    _close(got[0], want, 1e-15, "weighted heads over a sub-range")
    perm_pool = pool[::-1].copy()
    perm = np.array([1, 0], dtype=np.int32)
    got2 = O.dsa_index_scores(q, w2, perm_pool, perm, page_size=S, pos_begin=2, pos_end=7)
    assert np.array_equal(got, got2), "layout invariance"


def pin_topk_ties_and_order(O):
    """TopK equals a brute-force sort on (score descending, position
    ascending); equal scores go to the lower position; the result is in
    ascending position order; k >= n returns every position."""
    sc = np.array([[3.0, 1.0, 3.0, 2.0, 3.0, 0.5, 2.0]])
    assert O.topk_select(sc, 2).tolist() == [[0, 2]], "ties: lowest positions"
    assert O.topk_select(sc, 4).tolist() == [[0, 2, 3, 4]], "then the next score, lowest first"
    assert O.topk_select(sc, 10).tolist() == [list(range(7))], "k >= n: all"
    pos = np.array([40, 10, 30, 20, 50, 60, 70])
    assert O.topk_select(sc, 2, positions=pos).tolist() == [[30, 40]], "named positions"
    rng = np.random.default_rng(31)
    sc = rng.integers(-5, 6, (5, 300)).astype(np.float64)            # many ties
    for r in range(5):
        want = sorted(sorted(range(300), key=lambda j: (-sc[r, j], j))[:37])
        assert O.topk_select(sc[r:r + 1], 37)[0].tolist() == want, "brute force"


def pin_topk_local_candidates_merge(O):
    """Eq. glm-global-dsa: the top-k of the union of every shard's local top-k
    candidates (with their global positions) equals the global top-k; a
    shard's local selection alone (Eq. glm-local-dsa) generally does not."""
    rng = np.random.default_rng(32)
    sc = rng.integers(-20, 20, (4, 1000)).astype(np.float64)
    k = 50
    glob = O.topk_select(sc, k)
    bounds = [0, 137, 400, 401, 800, 1000]
    cand_pos, cand_sc = [], []
    for b, e in zip(bounds[:-1], bounds[1:]):
        loc = O.topk_select(sc[:, b:e], k) + b
        cand_pos.append(loc)
        cand_sc.append(np.take_along_axis(sc, loc, axis=1))
    cp, cs = np.concatenate(cand_pos, axis=1), np.concatenate(cand_sc, axis=1)
    merged = np.stack([O.topk_select(cs[r:r + 1], k, positions=cp[r])[0] for r in range(4)])
    assert np.array_equal(merged, glob), "candidate merge == global top-k"
    local0 = O.topk_select(sc[:, 0:137], k)
    assert not np.array_equal(local0, glob), "a local selection is not the global one"


ALL_PINS = [pin_single_key, pin_identical_keys, pin_zero_query, pin_scale_and_gqa,
            pin_merge_closed_form, pin_split_merge_invariance, pin_causal, pin_gather_bruteforce,
            pin_finite_differences, pin_bwd_partition, pin_torch_autograd, pin_sampled_rows,
            pin_sparse_full_index_is_dense, pin_sparse_subset, pin_sparse_invalid_entries, pin_decode, pin_bf16_round,
            pin_bf16_numerator_merge, pin_cyclic_ownership, pin_dsa_index_closed_form,
            pin_topk_ties_and_order, pin_topk_local_candidates_merge]
