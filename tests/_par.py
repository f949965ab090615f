"""Run the fp64 oracle over large inputs in a thread pool (test harness only).

The oracle computes each call from its definition with full score rows; at
2M keys one call would hold gigabytes of fp64 temporaries and run on one core.
These helpers split the keys into ranges and the rows into chunks, call the
oracle on each piece in a thread (BLAS limited to one thread per piece), and
compose the pieces with the oracle's own rules:

* forward ranges compose through ``O.lse_merge`` (Eq. qwen-lse-parts and
  qwen-global-attn; pinned: split + merge equals unsplit);
* dq contributions of a key partition add up (Eq. qwen-dq-reduce; pinned by the
  partition pin), and response dK/dV come from the response range alone;
* sparse rows are independent.
"""
from __future__ import annotations

import os
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle as O


def workers() -> int:
    return max(1, min(16, len(os.sched_getaffinity(0))))


def _pool_map(fn, items):
    """fn over items on the thread pool, in order; prints a line as each
    eighth of the pieces completes."""
    from concurrent.futures import as_completed
    from threadpoolctl import threadpool_limits
    items = list(items)
    t0 = time.perf_counter()
    with threadpool_limits(limits=1), ThreadPoolExecutor(max_workers=workers()) as ex:
        futs = {ex.submit(fn, it): i for i, it in enumerate(items)}
        res = [None] * len(items)
        step = max(1, len(items) // 8)
        for n, f in enumerate(as_completed(futs), 1):
            res[futs[f]] = f.result()
            if n % step == 0 or n == len(items):
                print(f"[oracle]   {n}/{len(items)} pieces, {time.perf_counter() - t0:.1f} s",
                      flush=True)
    return res


def key_ranges(begin, end, piece=65536):
    b = np.arange(begin, end, piece)
    return [(int(x), int(min(x + piece, end))) for x in b]


def _chunks(rows, n):
    rows = np.asarray(rows)
    return [c for c in np.array_split(rows, max(1, min(n, rows.size))) if c.size]


def dense_fwd(h, *, page_size, q_pos0, scale, rows, prefix_len, piece=65536, heads=None):
    """Full-row out and lse of ``rows`` (over every visible key; of the query
    heads ``heads`` only, when given): each chunk of rows is the merge of
    per-range oracle results over prefix ranges of ``piece`` keys and the
    response range."""
    rows = np.asarray(rows)
    kv_len = q_pos0 + h["q"].shape[0]
    ranges = key_ranges(0, prefix_len, piece) + [(prefix_len, kv_len)]
    n_chunks = max(1, (4 * workers()) // len(ranges))
    chunks = _chunks(rows, n_chunks)
    t0 = time.perf_counter()

    def one(task):
        r, c = task
        return O.attn_fwd(h["q"], h["k_pool"], h["v_pool"], h["page_table"], page_size=page_size,
                          q_pos0=q_pos0, scale=scale, kv_begin=r[0], kv_end=r[1], rows=c,
                          heads=heads)

    tasks = [(r, c) for c in chunks for r in ranges]
    parts = _pool_map(one, tasks)
    os_, ls_ = [], []
    for i in range(len(chunks)):
        p = parts[i * len(ranges):(i + 1) * len(ranges)]
        o, lse = O.lse_merge([x[0] for x in p], [x[1] for x in p])
        os_.append(o)
        ls_.append(lse)
    print(f"[oracle] dense fwd: {rows.size} rows x {kv_len} keys in {len(ranges)} ranges, "
          f"{time.perf_counter() - t0:.1f} s", flush=True)
    return np.concatenate(os_), np.concatenate(ls_, axis=1)


def dense_bwd(h, *, page_size, q_pos0, scale, prefix_len, rows, resp_keys, out, lse,
              piece=65536, resp_piece=512, kv_heads=None):
    """dq of ``rows`` over every visible key and the dK/dV of the response keys
    ``resp_keys``, given the oracle's full-row ``out``/``lse`` arrays ([R, Hq, Dv]
    / [Hq, R], filled at least for the rows that need them).  The keys are cut
    into prefix ranges of ``piece`` and response ranges of ``resp_piece``: dq is
    the sum of the ranges' contributions, and a response key's dK/dV come from
    the one range holding it (they depend only on that key's column of P and
    dS).  ``kv_heads`` restricts dq to those KV heads' query heads and dK/dV to
    those KV heads (oracle.attn_bwd)."""
    rows = np.asarray(rows, np.int64)
    assert np.all(np.diff(rows) > 0), "rows must be sorted and distinct"
    resp_keys = np.unique(np.asarray(resp_keys, np.int64))
    kv_len = q_pos0 + h["q"].shape[0]
    pre = key_ranges(0, prefix_len, piece)
    resp = key_ranges(prefix_len, kv_len, resp_piece)
    # prefix ranges hold no response key, so their dq rows split into chunks
    # (dq adds up over a row partition); a response range keeps every row,
    # since a key's dK/dV needs each row that sees it
    chunks = _chunks(rows, max(1, (4 * workers()) // max(1, len(pre))))
    tasks = [(r, c, False) for r in pre for c in chunks] + [(r, rows, True) for r in resp]
    t0 = time.perf_counter()
    kw = dict(page_size=page_size, prefix_len=prefix_len, q_pos0=q_pos0, scale=scale, out=out,
              lse=lse, kv_heads=kv_heads)

    def one(task):
        r, c, has_resp = task
        keys = resp_keys[(resp_keys >= r[0]) & (resp_keys < r[1])] if has_resp else resp_keys[:0]
        return O.attn_bwd(h["q"], h["k_pool"], h["v_pool"], h["page_table"], h["d_out"],
                          kv_begin=r[0], kv_end=r[1], resp_keys=keys, rows=c, **kw)

    parts = _pool_map(one, tasks)
    resp_parts = [p for p, t in zip(parts, tasks) if t[2]]
    dq = sum(p[0] for p in resp_parts) if resp_parts else None
    for p, (r, c, has_resp) in zip(parts, tasks):
        if has_resp:
            continue
        if dq is None:
            dq = np.zeros((rows.size,) + p[0].shape[1:])
        dq[np.searchsorted(rows, c)] += p[0]
    dk = np.concatenate([p[1] for p in resp_parts])
    dv = np.concatenate([p[2] for p in resp_parts])
    print(f"[oracle] dense bwd: {rows.size} dq rows, {resp_keys.size} response keys, "
          f"{time.perf_counter() - t0:.1f} s", flush=True)
    return dq, dk, dv


def sparse(h, *, page_size, prefix_len, q_pos0, scale, rows, backward=True, head_dim_v=512):
    """Sparse forward (and dq) of ``rows``, row chunks in parallel."""
    kw = dict(page_size=page_size, prefix_len=prefix_len, q_pos0=q_pos0, scale=scale,
              head_dim_v=head_dim_v)
    t0 = time.perf_counter()
    chunks = _chunks(rows, 4 * workers())

    def one(c):
        o, l = O.sparse_fwd(h["q"], h["latent_pool"], h["page_table"], h["idx"], rows=c, **kw)
        dq = (O.sparse_bwd(h["q"], h["latent_pool"], h["page_table"], h["idx"], h["d_out"],
                           rows=c, **kw) if backward else None)
        return o, l, dq

    parts = _pool_map(one, chunks)
    o = np.concatenate([p[0] for p in parts])
    lse = np.concatenate([p[1] for p in parts], axis=1)
    dq = np.concatenate([p[2] for p in parts]) if backward else None
    print(f"[oracle] sparse: {np.asarray(rows).size} rows in {time.perf_counter() - t0:.1f} s",
          flush=True)
    return o, lse, dq
