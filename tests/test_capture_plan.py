"""Split planning (CPU): capture chunk ranges and split plans cover every key
each chunk's rows can see, exactly once, and the page table hands every chunk
pages of its own; the blockwise forward's pieces tile the prefix and nest in
the backward's shard ranges."""
import numpy as np

from paper_2607_14952_amd import configs, inputs

SMALL = configs.CaptureConfig(name="cap_plan", seed=9, n_q_heads=4, n_kv_heads=2, head_dim=16,
                              page_size=64, length=5 * 512 + 77, chunk=512, keys_per_split=700)


def test_chunks_partition_the_prompt():
    cfg = SMALL
    r = [cfg.chunk_range(c) for c in range(cfg.n_chunks)]
    assert r[0][0] == 0 and r[-1][1] == cfg.length
    assert all(a[1] == b[0] for a, b in zip(r, r[1:]))
    assert r[-1][1] - r[-1][0] == 77


def test_splits_cover_earlier_keys_then_own():
    cfg = SMALL
    for c in range(cfg.n_chunks):
        b, e = cfg.chunk_range(c)
        sp = cfg.chunk_splits(c)
        assert sp[-1] == (b, e), "the chunk's own keys form the last split"
        flat = [k for s0, s1 in sp[:-1] for k in range(s0, s1)]
        assert flat == list(range(b)), "earlier keys covered once, in order"
        assert all(s1 - s0 <= cfg.keys_per_split for s0, s1 in sp[:-1])
    CAP = configs.CAPTURE_2M
    assert len(CAP.chunk_splits(CAP.n_chunks - 1)) == 65     # 64 x 32,704 earlier keys + own
    assert CAP.n_chunks == 512 and CAP.visible() == CAP.length * (CAP.length + 1) // 2


def test_chunks_get_pages_of_their_own():
    cfg = SMALL
    t = inputs.page_table(cfg)
    assert t.size == cfg.n_logical_pages and len(set(t.tolist())) == t.size
    assert t.min() >= 0 and t.max() < cfg.n_phys_pages


def test_capture_inputs_are_chunk_draws():
    cfg = SMALL
    h = inputs.capture_inputs(cfg)
    assert h["q_blocks"].shape == (cfg.n_chunks, cfg.chunk, 4, 16)
    assert h["k"].shape == (cfg.length, 2, 16) and h["v"].shape == (cfg.length, 2, 16)
    # a longer prompt with the same chunking keeps the earlier chunks' rows
    longer = inputs.capture_inputs(configs.CaptureConfig(**{**SMALL.__dict__, "length": 6 * 512}))
    assert np.array_equal(longer["k"][:5 * 512], h["k"][:5 * 512])


def test_blockwise_forward_plan():
    """c4's block forward: each of the 8 shard ranges cut 8 ways, contiguous,
    covering the prefix once, within one launch's split limit; the response
    split follows (its end moves with the block)."""
    cfg = configs.C4
    sp = cfg.splits()
    prefix = sp[:-1]
    assert len(prefix) == cfg.n_shards * cfg.splits_per_shard == 64
    assert prefix[0][0] == 0 and prefix[-1][1] == cfg.prefix_len
    assert all(a[1] == b[0] for a, b in zip(prefix, prefix[1:])), "contiguous"
    assert {e - b for b, e in prefix} == {cfg.prefix_len // 64}
    assert len(sp) <= 128
    # the backward's shard ranges are unions of consecutive forward pieces
    shard = cfg.prefix_len // cfg.n_shards
    for s in range(cfg.n_shards):
        pieces = prefix[8 * s:8 * s + 8]
        assert pieces[0][0] == s * shard and pieces[-1][1] == (s + 1) * shard
