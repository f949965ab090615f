"""Plain fp64 CPU oracle for response-replay attention.

TEST INFRASTRUCTURE ONLY.  Only the tests, the package smoke check and the
benchmark's CPU-baseline leg may import this module; the product path never
does.  It shares no code with the HIP library: every quantity is computed
here from its definition in the paper, in float64, with full score rows and
no online softmax, no tiling and no fusion.

Notation (paper, Sec. "Global Full-Attention Forward Composition"):
query row ``i`` of head ``h`` sits at logical position ``q_pos0 + i``; it sees
key position ``j`` iff ``j <= q_pos0 + i`` (the whole retained prefix plus the
response causally, diagonal included).  Head ``h`` reads KV head
``h // (Hq / Hkv)``.  Scores are ``s_ij = scale * q_i . k_j``.  A KV range
``[b, e)`` yields the normalized local output and natural-log normalizer of
Eq. qwen-local-attn; ranges compose through Eq. qwen-lse-parts and
Eq. qwen-global-attn.  Keys below ``prefix_len`` are stop-gradient state
(Eq. gradient-boundary): they feed dQ but get no dK/dV.
"""
from __future__ import annotations

import numpy as np


# --------------------------------------------------------------------------
# input decoding and the paged store
# --------------------------------------------------------------------------
def decode(x: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) or fp32 values -> float64."""
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return np.asarray(x, dtype=np.float64)


def gather(pool: np.ndarray, page_table: np.ndarray, page_size: int, positions) -> np.ndarray:
    """Rows of a paged store at logical ``positions`` (raw dtype, bit-exact).

    Logical position ``j`` lives in physical page ``page_table[j // S]`` at slot
    ``j % S`` (the logical-to-physical page map of Sec. "From Logical Shards to
    Physical Pages").  Returns ``[len(positions), Hkv, width]``."""
    positions = np.asarray(positions, dtype=np.int64)
    pages = page_table[positions // page_size].astype(np.int64)
    return pool[pages, positions % page_size]


def _kv(pool, page_table, page_size, positions, g, width=None):
    rows = gather(pool, page_table, page_size, positions)[:, g]
    if width is not None:
        rows = rows[:, :width]
    return decode(rows)


# --------------------------------------------------------------------------
# forward: Eq. qwen-local-attn over one KV range
# --------------------------------------------------------------------------
def attn_fwd(q, k_pool, v_pool, page_table, *, page_size, q_pos0, scale,
             kv_begin=0, kv_end=None, rows=None, heads=None, head_dim_v=None,
             row_block=64, key_positions=None):
    """Normalized output and log-normalizer of one KV range.

    Returns ``o [n_rows, n_heads, Dv]`` and ``lse [n_heads, n_rows]`` (natural
    log).  A row that sees no key of the range gets ``o = 0`` and
    ``lse = -inf``.  ``rows``/``heads`` select a subset (default: all).
    ``key_positions`` (sorted logical positions) replaces the range
    ``[kv_begin, kv_end)``: the key set of a shard that owns scattered pages."""
    R, Hq, D = q.shape
    Hkv = k_pool.shape[2]
    G = Hq // Hkv
    Dv = head_dim_v if head_dim_v is not None else v_pool.shape[3]
    rows = np.arange(R) if rows is None else np.asarray(rows)
    heads = np.arange(Hq) if heads is None else np.asarray(heads)
    if kv_end is None:
        kv_end = q_pos0 + R
    o = np.zeros((rows.size, heads.size, Dv))
    lse = np.full((heads.size, rows.size), -np.inf)
    last_visible = int(q_pos0 + rows.max()) + 1 if rows.size else kv_begin
    if key_positions is not None:
        keys = np.asarray(key_positions, dtype=np.int64)
        keys = keys[keys < last_visible] if rows.size else keys[:0]
    else:
        keys = np.arange(kv_begin, min(kv_end, last_visible))
    if keys.size == 0 or rows.size == 0:
        return o, lse
    for g in sorted({int(h) // G for h in heads}):
        K = _kv(k_pool, page_table, page_size, keys, g)
        V = _kv(v_pool, page_table, page_size, keys, g, Dv)
        for hi_, h in enumerate(heads):
            if int(h) // G != g:
                continue
            for r0 in range(0, rows.size, row_block):
                rr = rows[r0:r0 + row_block]
                Q = decode(q[rr, h])
                s = scale * (Q @ K.T)
                visible = keys[None, :] <= (q_pos0 + rr)[:, None]
                s = np.where(visible, s, -np.inf)
                m = s.max(axis=1)
                any_vis = np.isfinite(m)
                m_safe = np.where(any_vis, m, 0.0)
                w = np.exp(s - m_safe[:, None])          # 0 where masked
                z = w.sum(axis=1)
                ell = np.where(any_vis, m_safe + np.log(np.where(any_vis, z, 1.0)), -np.inf)
                p = np.where(any_vis[:, None], w / np.where(any_vis, z, 1.0)[:, None], 0.0)
                o[r0:r0 + rr.size, hi_] = p @ V
                lse[hi_, r0:r0 + rr.size] = ell
    return o, lse


def _merge_weights(lse_parts):
    """Shared part of Eq. qwen-lse-parts / qwen-global-attn: the part weights
    e^(l_r - m) with m = max_r l_r (0 for empty parts), a = sum of the weights
    (1 where every part is empty) and l = m + log a (-inf there)."""
    L = np.stack([np.asarray(x, dtype=np.float64) for x in lse_parts])      # [S, H, R]
    m = L.max(axis=0)
    alive = np.isfinite(m)
    m_safe = np.where(alive, m, 0.0)
    w = np.where(np.isfinite(L), np.exp(L - m_safe[None]), 0.0)             # [S, H, R]
    a = w.sum(axis=0)
    a_safe = np.where(alive, a, 1.0)
    lse = np.where(alive, m_safe + np.log(a_safe), -np.inf)
    return w, a_safe, lse


def lse_merge(o_parts, lse_parts):
    """Compose range results (Eq. qwen-lse-parts, Eq. qwen-global-attn).

    ``o_parts``: list of ``[R, H, Dv]``; ``lse_parts``: list of ``[H, R]``.
    m = max_r l_r;  a = sum_r e^(l_r - m);  n = sum_r e^(l_r - m) o_r;
    o = n / a;  l = m + log a.  Ranges with l_r = -inf carry weight 0; a row whose
    every range is empty stays o = 0, l = -inf."""
    w, a_safe, lse = _merge_weights(lse_parts)
    O = np.stack([np.asarray(x, dtype=np.float64) for x in o_parts])        # [S, R, H, Dv]
    n = np.einsum("shr,srhd->rhd", w, O)
    o = n / a_safe.T[:, :, None]
    return o, lse


def bf16_round(x):
    """Nearest bfloat16 value (ties to even) of each float64 in ``x``, as float64.

    bfloat16 keeps 8 significant bits and float32's exponent range.  Written
    from that definition: x = m 2^e with 0.5 <= |m| < 1, and m 2^8 is rounded
    to an integer, ties to even (normal range only, which is all this oracle
    meets; zero stays zero)."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)


def lse_merge_bf16_numerator(o_parts, lse_parts):
    """Eq. qwen-lse-parts / qwen-global-attn with the numerator reduced in
    bf16, the production composition described right after Eq.
    qwen-global-attn: m, a and l are exact; each part's numerator term
    e^(l_r - m) o_r is rounded to bf16, and the terms are summed in part order
    with the running sum rounded to bf16 after every addition; o = n / a.
    (The order and the rounding of each term are this oracle's reading of a
    bf16 all-reduce.)"""
    w, a_safe, lse = _merge_weights(lse_parts)
    n = None
    for r, o_r in enumerate(o_parts):
        term = bf16_round(w[r].T[:, :, None] * np.asarray(o_r, dtype=np.float64))
        n = term if n is None else bf16_round(n + term)
    return n / a_safe.T[:, :, None], lse


# --------------------------------------------------------------------------
# block-cyclic page ownership (Sec. "From Logical Shards to Physical Pages")
# --------------------------------------------------------------------------
def cyclic_owned_positions(prefix_len, page_size, n_shards, shard):
    """Logical prefix positions of shard ``shard`` when logical page p is owned
    by shard p mod n_shards (Eq. qwen-page-owner), in increasing order."""
    n_pages = -(-prefix_len // page_size)
    pages = np.arange(shard, n_pages, n_shards, dtype=np.int64)
    pos = (pages[:, None] * page_size + np.arange(page_size)[None, :]).reshape(-1)
    return pos[pos < prefix_len]


# --------------------------------------------------------------------------
# backward: exact attention gradients with the prefix held as stop-gradient
# --------------------------------------------------------------------------
def attn_bwd(q, k_pool, v_pool, page_table, d_out, *, page_size, prefix_len, q_pos0, scale,
             kv_begin=0, kv_end=None, out=None, lse=None, rows=None, resp_keys=None,
             head_dim_v=None, row_block=64, kv_heads=None):
    """Gradients of L = sum(d_out * O) where O is the full replay output.

    * ``dq [n_rows, Hq, D]``: contribution of the keys in ``[kv_begin, kv_end)``
      (Eq. qwen-dq-reduce: summing the contributions of a partition of the keys
      gives the full dq);
    * ``dk_resp, dv_resp [n_resp_keys, Hkv, D|Dv]``: gradients of the response keys
      ``resp_keys`` (default: every response key in the range), i.e. positions
      ``>= prefix_len``; prefix keys get none (Eq. gradient-boundary).

    ``out``/``lse`` are the full forward over every visible key for all rows
    (computed here in fp64 when not given).  ``rows`` restricts dq to a subset of
    rows; dk/dv always use every row that sees the key.  ``kv_heads`` restricts
    the computation to those KV heads and the query heads of their groups: dq
    then holds those query heads (in order) and dk/dv those KV heads.  A KV
    head's gradient sums over its own group only, so its dk/dv are complete."""
    R, Hq, D = q.shape
    Hkv = k_pool.shape[2]
    G = Hq // Hkv
    Dv = head_dim_v if head_dim_v is not None else v_pool.shape[3]
    kv_len = q_pos0 + R
    if kv_end is None:
        kv_end = kv_len
    kv_end = min(kv_end, kv_len)
    dq_rows = np.arange(R) if rows is None else np.asarray(rows)
    if resp_keys is None:
        resp_keys = np.arange(max(kv_begin, prefix_len), max(kv_end, prefix_len))
    resp_keys = np.asarray(resp_keys, dtype=np.int64)
    assert np.all((resp_keys >= prefix_len) & (resp_keys >= kv_begin) & (resp_keys < kv_end))

    # rows whose forward state is needed: dq rows, and every row that sees a resp key
    need = set(dq_rows.tolist())
    if resp_keys.size:
        need.update(range(int(resp_keys.min()) - q_pos0, R))
    need_rows = np.array(sorted(need), dtype=np.int64)
    if out is None or lse is None:
        o_n, l_n = attn_fwd(q, k_pool, v_pool, page_table, page_size=page_size, q_pos0=q_pos0,
                            scale=scale, rows=need_rows, head_dim_v=Dv)
        row_at = {int(r): k for k, r in enumerate(need_rows)}
    else:
        o_n, l_n = np.asarray(out, np.float64)[need_rows], np.asarray(lse, np.float64)[:, need_rows]
        row_at = {int(r): k for k, r in enumerate(need_rows)}
    dO_all = decode(d_out)
    # Delta_ih = dO_ih . o_ih  (the oracle's own fp64 output)
    delta = np.einsum("rhd,rhd->hr", dO_all[need_rows], o_n)

    kvh = np.arange(Hkv) if kv_heads is None else np.asarray(kv_heads)
    dq = np.zeros((dq_rows.size, kvh.size * G, D))
    dk = np.zeros((resp_keys.size, kvh.size, D))
    dv = np.zeros((resp_keys.size, kvh.size, Dv))
    keys = np.arange(kv_begin, kv_end)
    resp_col = resp_keys - kv_begin                     # columns of the range holding resp keys
    for gi, g in enumerate(kvh):
        K = _kv(k_pool, page_table, page_size, keys, g)
        V = _kv(v_pool, page_table, page_size, keys, g, Dv)
        for h in range(g * G, (g + 1) * G):
            hl = gi * G + h - g * G                     # this head's slot in dq
            for r0 in range(0, need_rows.size, row_block):
                rr = need_rows[r0:r0 + row_block]
                idx = np.array([row_at[int(r)] for r in rr])
                Q = decode(q[rr, h])
                dO = dO_all[rr, h]
                s = scale * (Q @ K.T)
                visible = keys[None, :] <= (q_pos0 + rr)[:, None]
                ell = l_n[h, idx]
                P = np.where(visible, np.exp(np.where(visible, s, 0.0) - ell[:, None]), 0.0)
                dP = dO @ V.T
                dS = P * (dP - delta[h, idx][:, None])
                # dq for the requested rows
                sel = np.isin(rr, dq_rows)
                if sel.any():
                    pos = np.searchsorted(dq_rows, rr[sel])
                    dq[pos, hl] += scale * (dS[sel] @ K)
                if resp_keys.size:
                    dk[:, gi] += scale * (dS[:, resp_col].T @ Q)
                    dv[:, gi] += P[:, resp_col].T @ dO
    return dq, dk, dv


# --------------------------------------------------------------------------
# sparse latent replay: Eq. dsa-attention over the selected prefix positions
# --------------------------------------------------------------------------
def _sparse_visible(idx_row, prefix_len, pos):
    """Selected prefix positions, then the response positions up to ``pos``.

    Eq. dsa-attention draws the selection from the prefix only.  An entry
    outside ``[0, prefix_len)`` selects no key: the top-k pads a row that has
    fewer than k candidates with -1, and a position at or past the prefix is
    already in the response window."""
    sel = np.asarray(idx_row, np.int64)
    sel = sel[(sel >= 0) & (sel < prefix_len)]
    return np.concatenate([sel, np.arange(prefix_len, pos + 1)])


def sparse_fwd(q, latent_pool, page_table, idx, *, page_size, prefix_len, q_pos0, scale,
               head_dim_v, rows=None):
    """MLA/DSA replay: every head of row ``t`` attends to the latent rows
    ``c_s`` for ``s`` in its selected prefix positions plus the response positions
    ``prefix_len <= s <= q_pos0 + t``; keys are all ``Dk`` channels of ``c_s`` and
    values its first ``Dv`` channels (absorbed MLA, Sec. "Layer Anatomy: MLA/DSA").
    Returns ``o [n_rows, H, Dv]``, ``lse [H, n_rows]``."""
    R, H, Dk = q.shape
    rows = np.arange(R) if rows is None else np.asarray(rows)
    o = np.zeros((rows.size, H, head_dim_v))
    lse = np.zeros((H, rows.size))
    for k_, t in enumerate(rows):
        keys = _sparse_visible(idx[t], prefix_len, q_pos0 + int(t))
        C = _kv(latent_pool, page_table, page_size, keys, 0)
        Q = decode(q[t])                                   # [H, Dk]
        s = scale * (Q @ C.T)                              # [H, n]
        m = s.max(axis=1)
        w = np.exp(s - m[:, None])
        z = w.sum(axis=1)
        o[k_] = (w / z[:, None]) @ C[:, :head_dim_v]
        lse[:, k_] = m + np.log(z)
    return o, lse


def sparse_bwd(q, latent_pool, page_table, idx, d_out, *, page_size, prefix_len, q_pos0,
               scale, head_dim_v, rows=None):
    """dq of L = sum(d_out * O) for the sparse replay (latent rows get no gradient)."""
    R, H, Dk = q.shape
    rows = np.arange(R) if rows is None else np.asarray(rows)
    dq = np.zeros((rows.size, H, Dk))
    for k_, t in enumerate(rows):
        keys = _sparse_visible(idx[t], prefix_len, q_pos0 + int(t))
        C = _kv(latent_pool, page_table, page_size, keys, 0)
        Q = decode(q[t])
        dO = decode(d_out[t])                              # [H, Dv]
        s = scale * (Q @ C.T)
        m = s.max(axis=1)
        w = np.exp(s - m[:, None])
        P = w / w.sum(axis=1)[:, None]
        o = P @ C[:, :head_dim_v]
        delta = (dO * o).sum(axis=1)
        dP = dO @ C[:, :head_dim_v].T
        dS = P * (dP - delta[:, None])
        dq[k_] = scale * (dS @ C)
    return dq


# --------------------------------------------------------------------------
# DSA index selection (Eq. dsa-index, Eq. glm-global-dsa)
# --------------------------------------------------------------------------
def dsa_index_scores(q_index, w_index, k_index_pool, page_table, *, page_size, pos_begin,
                     pos_end, rows=None):
    """Index scores of Eq. dsa-index: I[t, s] = sum_j w[t, j] ReLU(<q[t, j], k_s>)
    for rows t and prefix positions s in [pos_begin, pos_end).

    ``q_index`` [R, H_I, d] and ``k_index_pool`` [n_phys, S, d] (bf16 bit
    patterns or floats; one index key per position, shared by the heads),
    ``w_index`` [R, H_I].  Returns ``[n_rows, pos_end - pos_begin]`` float64."""
    R = q_index.shape[0]
    rows = np.arange(R) if rows is None else np.asarray(rows)
    K = decode(gather(k_index_pool, page_table, page_size, np.arange(pos_begin, pos_end)))
    out = np.zeros((rows.size, pos_end - pos_begin))
    for k_, t in enumerate(rows):
        Q = decode(q_index[t])                              # [H_I, d]
        W = np.asarray(w_index[t], dtype=np.float64)        # [H_I]
        out[k_] = W @ np.maximum(Q @ K.T, 0.0)
    return out


def topk_select(scores, k, positions=None):
    """TopK of Eq. dsa-attention / glm-global-dsa for each row of ``scores``
    [rows, n]: the k largest scores, equal scores ordered by lower position
    first (the deterministic rule of a candidate merge), returned as positions
    in ascending order ([rows, min(k, n)] int64).  ``positions`` [n] or
    [rows, n] names each column's position (default 0 .. n - 1)."""
    scores = np.asarray(scores, dtype=np.float64)
    rows, n = scores.shape
    pos = np.broadcast_to(np.arange(n) if positions is None else np.asarray(positions),
                          (rows, n))
    take = min(k, n)
    out = np.empty((rows, take), dtype=np.int64)
    for r in range(rows):
        order = np.lexsort((pos[r], -scores[r]))            # by score desc, then position asc
        out[r] = np.sort(pos[r][order[:take]])
    return out
