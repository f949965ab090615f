"""The seeded input generator: deterministic, right shapes, valid tables."""
import numpy as np

from paper_2607_14952_amd import configs, inputs


def test_c1_shapes_and_determinism():
    c = configs.C1
    a = inputs.dense_inputs(c)
    b = inputs.dense_inputs(c)
    assert a["q"].shape == (128, 2, 64) and a["q"].dtype == np.float32
    assert a["k_pool"].shape == (c.n_phys_pages, 64, 1, 64)
    assert np.array_equal(a["page_table"], np.arange(c.n_logical_pages))
    for k in ("q", "k_pool", "v_pool", "d_out"):
        assert np.array_equal(a[k], b[k])


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1.0 + 2 ** -8 + 2 ** -10],
                 dtype=np.float32)
    got = inputs.bf16_bits_to_f32(inputs.to_bf16_bits(x))
    # ties go to the even mantissa; above-half rounds up
    assert got.tolist() == [1.0, 1.0, 1.0 + 2 ** -6, -2.5, 1.0 + 2 ** -7]


def test_tables_are_injective():
    for name, table in (("perm", "perm"), ("sample", "sample")):
        c = configs.C3.scaled(prefix_len=16384, resp_len=512, table=table, pool_slack=1.25)
        t = inputs.page_table(c)
        assert t.size == c.n_logical_pages
        assert np.unique(t).size == t.size and t.min() >= 0 and t.max() < c.n_phys_pages


def test_planted_keys_raise_target_score():
    c = configs.C3.scaled(prefix_len=8192, resp_len=64, plant_frac=0.01)
    d = inputs.dense_inputs(c, with_dout=False)
    pos, rows, heads = d["planted"]
    assert pos.size == 82 and np.all(np.diff(pos) > 0)
    q = inputs.bf16_bits_to_f32(d["q"]).astype(np.float64)
    pt = d["page_table"]
    for j, t, h in list(zip(pos, rows, heads))[:8]:
        k = inputs.bf16_bits_to_f32(d["k_pool"][pt[j // 256], j % 256, h // 8]).astype(np.float64)
        assert q[t, h] @ k / 16.0 > 40.0


def test_sparse_indices_sorted_unique():
    c = configs.C5.scaled(prefix_len=4096, resp_len=16, topk=256)
    idx = inputs.sparse_indices(c)
    assert idx.shape == (16, 256)
    assert np.all(np.diff(idx, axis=1) > 0) and idx.min() >= 0 and idx.max() < 4096
