"""Seeded synthetic inputs for response-replay attention.

This module only draws random numbers and lays them out; it computes nothing
of the attention method.  Both the HIP path and the CPU oracle read the bytes
it produces, so the two always see identical inputs.

Recipe (all draws fp32 from numpy's PCG64, bf16 configs rounded to nearest-even):

* streams: 0 page table, 1 K pool, 2 V pool, 3 Q, 4 dO, 5 planted keys, 6 sparse indices;
* every physical KV page ``p`` is drawn from ``SeedSequence([seed, stream, p])`` so
  pages can be generated in parallel and independently of the pool size;
* Q and dO are drawn in chunks of 2**20 values from ``SeedSequence([seed, stream, chunk])``;
* page table: identity, a seeded permutation of all logical pages, or (``sample``) a
  seeded sample without replacement from a pool with free pages;
* planted keys: a fraction of prefix positions ``j`` each picks a target query row ``t`` and
  head ``h`` and gets ``k[j, h // G] += gain * q[t, h]`` before rounding, which raises that
  one score by about ``gain * sqrt(D)`` and makes the per-shard log-normalizers differ by
  tens of nats;
* sparse replay: each query row draws ``topk`` distinct prefix positions, sorted ascending.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

STREAM_TABLE, STREAM_K, STREAM_V, STREAM_Q, STREAM_DO, STREAM_PLANT, STREAM_IDX, STREAM_PARTS, \
    STREAM_IQ, STREAM_IW, STREAM_IK = range(11)
_CHUNK = 1 << 20


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key))))


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even) and return the raw 16-bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    out = np.empty(x.shape, dtype=np.uint16)
    flat_u, flat_o = u.reshape(-1), out.reshape(-1)

    def work(lo, hi):
        v = flat_u[lo:hi]
        flat_o[lo:hi] = ((v + np.uint32(0x7FFF) + ((v >> np.uint32(16)) & np.uint32(1)))
                         >> np.uint32(16)).astype(np.uint16)

    n = flat_u.size
    step = max(_CHUNK, -(-n // _threads()))
    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(lambda lo: work(lo, min(n, lo + step)), range(0, n, step)))
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal_chunks(seed: int, stream: int, n: int) -> np.ndarray:
    """n standard normals, chunk c drawn from SeedSequence([seed, stream, c])."""
    out = np.empty(n, dtype=np.float32)

    def fill(c):
        lo = c * _CHUNK
        hi = min(n, lo + _CHUNK)
        _rng(seed, stream, c).standard_normal(hi - lo, dtype=np.float32, out=out[lo:hi])

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(fill, range(-(-n // _CHUNK))))
    return out


def page_table(cfg, n_logical: int | None = None) -> np.ndarray:
    """Logical page -> physical page id (int32)."""
    n_logical = cfg.n_logical_pages if n_logical is None else n_logical
    rng = _rng(cfg.seed, STREAM_TABLE)
    if cfg.table == "identity":
        t = np.arange(n_logical)
    elif cfg.table == "perm":
        t = rng.permutation(cfg.n_phys_pages)[:n_logical]
    elif cfg.table == "sample":
        t = rng.choice(cfg.n_phys_pages, size=n_logical, replace=False)
    else:
        raise ValueError(cfg.table)
    return t.astype(np.int32)


def _pool(cfg, stream: int, width: int, n_heads: int, plants=None) -> np.ndarray:
    """Physical pool [n_phys, S, n_heads, width] filled page by page.

    ``plants`` maps physical page -> list of (slot, head, fp32 vector) additions made
    before rounding."""
    S = cfg.page_size
    per_page = S * n_heads * width
    bf16 = cfg.dtype == "bf16"
    out = np.empty((cfg.n_phys_pages, S, n_heads, width), dtype=np.uint16 if bf16 else np.float32)

    def fill(p):
        x = _rng(cfg.seed, stream, p).standard_normal(per_page, dtype=np.float32)
        x = x.reshape(S, n_heads, width)
        if plants is not None and p in plants:
            for slot, g, vec in plants[p]:
                x[slot, g] += vec
        if bf16:
            u = x.view(np.uint32)
            out[p] = ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))
                      >> np.uint32(16)).astype(np.uint16)
        else:
            out[p] = x

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(fill, range(cfg.n_phys_pages)))
    return out


def _dense_tensor(cfg, stream: int, shape) -> np.ndarray:
    x = normal_chunks(cfg.seed, stream, int(np.prod(shape))).reshape(shape)
    return to_bf16_bits(x) if cfg.dtype == "bf16" else x


def plant_targets(cfg, q_f32: np.ndarray, table: np.ndarray):
    """Planted prefix keys: returns (positions, target rows, target heads) and the
    per-physical-page additions used while drawing the K pool."""
    n = int(round(cfg.plant_frac * cfg.prefix_len))
    if n == 0:
        return None, None
    rng = _rng(cfg.seed, STREAM_PLANT)
    pos = np.sort(rng.choice(cfg.prefix_len, size=n, replace=False))
    rows = rng.integers(0, cfg.resp_len, size=n)
    heads = rng.integers(0, cfg.n_q_heads, size=n)
    plants: dict[int, list] = {}
    for j, t, h in zip(pos.tolist(), rows.tolist(), heads.tolist()):
        p = int(table[j // cfg.page_size])
        d = q_f32[t, h]
        if cfg.plant_unit:   # the score-sigma variant: a unit direction
            d = d / np.float32(np.linalg.norm(d))
        plants.setdefault(p, []).append((j % cfg.page_size, h // cfg.group, cfg.plant_gain * d))
    return (pos, rows, heads), plants


def dense_inputs(cfg, with_dout: bool = True) -> dict:
    """q [R,Hq,D], k_pool/v_pool [n_phys,S,Hkv,D|Dv], page_table [n_logical], d_out [R,Hq,Dv].

    bf16 tensors are returned as uint16 bit patterns, fp32 ones as float32."""
    R, Hq, Hkv = cfg.resp_len, cfg.n_q_heads, cfg.n_kv_heads
    table = page_table(cfg)
    q = _dense_tensor(cfg, STREAM_Q, (R, Hq, cfg.head_dim))
    q_f32 = bf16_bits_to_f32(q) if cfg.dtype == "bf16" else q
    planted, plants = plant_targets(cfg, q_f32, table)
    k_pool = _pool(cfg, STREAM_K, cfg.head_dim, Hkv, plants)
    v_pool = _pool(cfg, STREAM_V, cfg.head_dim_v, Hkv)
    out = dict(q=q, k_pool=k_pool, v_pool=v_pool, page_table=table, planted=planted)
    if with_dout:
        out["d_out"] = _dense_tensor(cfg, STREAM_DO, (R, Hq, cfg.head_dim_v))
    return out


def sparse_indices(cfg) -> np.ndarray:
    """[R, topk] int32: per query row, topk distinct prefix positions in ascending order."""
    R, k, P = cfg.resp_len, cfg.topk, cfg.prefix_len
    if k > P:
        raise ValueError("topk exceeds the prefix")
    out = np.empty((R, k), dtype=np.int32)

    def fill(t):
        rng = _rng(cfg.seed, STREAM_IDX, t)
        got = np.empty(0, dtype=np.int64)
        while got.size < k:
            extra = rng.integers(0, P, size=k + 64)
            got = np.unique(np.concatenate([got, extra]))
        sel = rng.choice(got.size, size=k, replace=False)
        out[t] = np.sort(got[sel])

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(fill, range(R)))
    return out


def sparse_inputs(cfg, with_dout: bool = True) -> dict:
    """q [R,H,Dk], latent_pool [n_phys,S,1,Dk] (keys = all Dk channels, values = the
    first Dv), page_table, idx [R,topk], d_out [R,H,Dv]."""
    R, H = cfg.resp_len, cfg.n_q_heads
    table = page_table(cfg)
    q = _dense_tensor(cfg, STREAM_Q, (R, H, cfg.head_dim))
    latent = _pool(cfg, STREAM_K, cfg.head_dim, 1)
    out = dict(q=q, latent_pool=latent, page_table=table, idx=sparse_indices(cfg))
    if with_dout:
        out["d_out"] = _dense_tensor(cfg, STREAM_DO, (R, H, cfg.head_dim_v))
    if cfg.index_heads:
        # index queries, head weights and one 128-wide index key per position in
        # pages parallel to the latent pages (same table)
        Hi = cfg.index_heads
        out["q_index"] = to_bf16_bits(
            _rng(cfg.seed, STREAM_IQ).standard_normal((R, Hi, 128), dtype=np.float32))
        out["w_index"] = (_rng(cfg.seed, STREAM_IW).standard_normal((R, Hi), dtype=np.float32)
                          / np.float32(np.sqrt(Hi)))
        out["k_index_pool"] = to_bf16_bits(normal_chunks(
            cfg.seed, STREAM_IK, cfg.n_phys_pages * cfg.page_size * 128).reshape(
                cfg.n_phys_pages, cfg.page_size, 128))
    return out


# ---------------------------------------------------------------- resident prefix + responses
def member_seed(cfg, member: int) -> int:
    """Seed of response `member` replayed against a shared prefix (config seed s -> 1000*s + m)."""
    return 1000 * cfg.seed + member


def prefix_store(cfg) -> dict:
    """Pools [n_phys, S, Hkv, D|Dv] and the prefix part of the page table
    ([n_prefix_pages] int32); physical pages not named by it form the free list
    (ascending) from which response pages are appended."""
    table = page_table(cfg, n_logical=cfg.n_prefix_pages)
    k_pool = _pool(cfg, STREAM_K, cfg.head_dim, cfg.n_kv_heads)
    v_pool = _pool(cfg, STREAM_V, cfg.head_dim_v, cfg.n_kv_heads)
    used = np.zeros(cfg.n_phys_pages, dtype=bool)
    used[table] = True
    return dict(k_pool=k_pool, v_pool=v_pool, prefix_table=table,
                free_pages=np.flatnonzero(~used).astype(np.int32))


def response_inputs(cfg, member: int) -> dict:
    """One response branch: q [R,Hq,D], its own K/V rows k [R,Hkv,D], v [R,Hkv,Dv]
    and d_out [R,Hq,Dv], drawn from the member's seed."""
    s = member_seed(cfg, member)
    R = cfg.resp_len

    def draw(stream, shape):
        x = normal_chunks(s, stream, int(np.prod(shape))).reshape(shape)
        return to_bf16_bits(x) if cfg.dtype == "bf16" else x

    return dict(q=draw(STREAM_Q, (R, cfg.n_q_heads, cfg.head_dim)),
                k=draw(STREAM_K, (R, cfg.n_kv_heads, cfg.head_dim)),
                v=draw(STREAM_V, (R, cfg.n_kv_heads, cfg.head_dim_v)),
                d_out=draw(STREAM_DO, (R, cfg.n_q_heads, cfg.head_dim_v)))


def merge_parts(seed: int, n_parts: int, n_q: int, n_heads: int, dv: int,
                empty_frac: float = 0.05):
    """Partial results to compose: o [n_parts, n_q, n_heads, dv] fp32 standard
    normals and lse [n_parts, n_heads, n_q] fp32 normals of spread 3, with a
    fraction of (part, head, row) entries empty (lse = -inf, o = 0), and (with
    at least 3 rows) one row empty in every part."""
    rng = _rng(seed, STREAM_PARTS)
    o = rng.standard_normal((n_parts, n_q, n_heads, dv), dtype=np.float32)
    lse = (3.0 * rng.standard_normal((n_parts, n_heads, n_q))).astype(np.float32)
    empty = rng.random((n_parts, n_heads, n_q)) < empty_frac
    if n_q >= 3:
        empty[:, :, n_q // 2] = True
    lse[empty] = -np.inf
    o[np.transpose(empty, (0, 2, 1))] = 0.0
    return o, lse


def capture_inputs(cfg) -> dict:
    """Prompt rows for a chunked capture: q_blocks [n_q_blocks, chunk, Hq, D]
    (block b from stream (seed, Q, b)), k and v [length, Hkv, D] (chunk c's rows
    from streams (seed, K|V, c)), all bf16 bit patterns, and the page table.
    Chunk c's queries are the first rows of block c mod n_q_blocks."""
    Hq, Hkv, D, C = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.chunk

    def block(stream, key, rows, heads):
        x = _rng(cfg.seed, stream, key).standard_normal((rows, heads, D), dtype=np.float32)
        return to_bf16_bits(x)

    with ThreadPoolExecutor(_threads()) as ex:
        qb = list(ex.map(lambda b: block(STREAM_Q, b, C, Hq), range(cfg.n_q_blocks)))
        rows = [cfg.chunk_range(c) for c in range(cfg.n_chunks)]
        ks = list(ex.map(lambda c: block(STREAM_K, c, rows[c][1] - rows[c][0], Hkv),
                         range(cfg.n_chunks)))
        vs = list(ex.map(lambda c: block(STREAM_V, c, rows[c][1] - rows[c][0], Hkv),
                         range(cfg.n_chunks)))
    return {"q_blocks": np.stack(qb), "k": np.concatenate(ks), "v": np.concatenate(vs),
            "page_table": page_table(cfg)}


def dsa_index_inputs(seed: int, n_q: int, n_heads: int, n_pos: int, page_size: int,
                     head_dim: int = 128, pool_slack: float = 1.25) -> dict:
    """Index-selection inputs (Eq. dsa-index): q_index [n_q, n_heads, head_dim]
    and one index key per position in a paged pool [n_phys, page_size,
    head_dim] (bf16 bit patterns, N(0,1) before rounding), head weights
    w_index [n_q, n_heads] fp32 N(0,1) / sqrt(n_heads), and a page table
    (seeded choice of distinct physical pages)."""
    n_log = -(-n_pos // page_size)
    n_phys = max(n_log, int(np.ceil(n_log * pool_slack)))
    q = _rng(seed, STREAM_IQ).standard_normal((n_q, n_heads, head_dim), dtype=np.float32)
    w = (_rng(seed, STREAM_IW).standard_normal((n_q, n_heads), dtype=np.float32)
         / np.float32(np.sqrt(n_heads)))
    k = normal_chunks(seed, STREAM_IK, n_phys * page_size * head_dim).reshape(
        n_phys, page_size, head_dim)
    table = _rng(seed, STREAM_TABLE).choice(n_phys, size=n_log, replace=False).astype(np.int32)
    return {"q_index": to_bf16_bits(q), "w_index": w, "k_index_pool": to_bf16_bits(k),
            "page_table": table}
