"""Plant plausible mistakes in copies of the oracle (on the CPU) and check that
each one trips at least one pin, so the pins are not vacuous."""
import os
import types

import pytest

from tests._pins import ALL_PINS

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "attention.py")

# (name, text in the oracle, replacement)
MUTATIONS = [
    ("causal_exclusive", "visible = keys[None, :] <= (q_pos0 + rr)[:, None]\n                s = np.where",
     "visible = keys[None, :] < (q_pos0 + rr)[:, None]\n                s = np.where"),
    ("no_scale_fwd", "s = scale * (Q @ K.T)\n                visible = keys[None, :] <= (q_pos0 + rr)[:, None]\n                s = np.where",
     "s = (Q @ K.T)\n                visible = keys[None, :] <= (q_pos0 + rr)[:, None]\n                s = np.where"),
    ("gqa_modulo", "if int(h) // G != g:", "if int(h) % Hkv != g:"),
    ("gqa_modulo_set", "sorted({int(h) // G for h in heads})", "sorted({int(h) % Hkv for h in heads})"),
    ("lse_log2", "ell = np.where(any_vis, m_safe + np.log(", "ell = np.where(any_vis, m_safe + np.log2("),
    ("lse_no_max", "ell = np.where(any_vis, m_safe + np.log(", "ell = np.where(any_vis, 0.0 + np.log("),
    ("merge_no_shift", "lse = np.where(alive, m_safe + np.log(a_safe), -np.inf)",
     "lse = np.where(alive, np.log(a_safe), -np.inf)"),
    ("merge_unnormalized", "o = n / a_safe.T[:, :, None]", "o = n"),
    ("merge_plain_mean", "w = np.where(np.isfinite(L), np.exp(L - m_safe[None]), 0.0)",
     "w = np.where(np.isfinite(L), 1.0, 0.0)"),
    ("table_ignored", "pages = page_table[positions // page_size].astype(np.int64)",
     "pages = (positions // page_size).astype(np.int64)"),
    ("bwd_no_delta", "dS = P * (dP - delta[h, idx][:, None])", "dS = P * dP"),
    ("bwd_dq_no_scale", "dq[pos, hl] += scale * (dS[sel] @ K)", "dq[pos, hl] += (dS[sel] @ K)"),
    ("bwd_dv_uses_dS", "dv[:, gi] += P[:, resp_col].T @ dO", "dv[:, gi] += dS[:, resp_col].T @ dO"),
    ("bwd_dk_uses_P", "dk[:, gi] += scale * (dS[:, resp_col].T @ Q)", "dk[:, gi] += scale * (P[:, resp_col].T @ Q)"),
    ("bwd_resp_shift", "resp_col = resp_keys - kv_begin", "resp_col = resp_keys - kv_begin - 1"),
    ("bwd_P_no_lse", "np.exp(np.where(visible, s, 0.0) - ell[:, None])", "np.exp(np.where(visible, s, 0.0))"),
    ("bwd_delta_dO_sq", 'delta = np.einsum("rhd,rhd->hr", dO_all[need_rows], o_n)',
     'delta = np.einsum("rhd,rhd->hr", dO_all[need_rows], dO_all[need_rows])'),
    ("sparse_window_exclusive", "np.arange(prefix_len, pos + 1)", "np.arange(prefix_len, pos)"),
    ("sparse_values_tail", "o[k_] = (w / z[:, None]) @ C[:, :head_dim_v]",
     "o[k_] = (w / z[:, None]) @ C[:, -head_dim_v:]"),
    ("sparse_dq_no_delta", "dS = P * (dP - delta[:, None])\n        dq[k_]", "dS = P * dP\n        dq[k_]"),
    ("sparse_pads_clamped", "sel = sel[(sel >= 0) & (sel < prefix_len)]",
     "sel = np.clip(sel, 0, prefix_len - 1)"),
    ("sparse_pads_kept_past_prefix", "sel = sel[(sel >= 0) & (sel < prefix_len)]", "sel = sel[sel >= 0]"),
    ("decode_shift_15", "return (x.astype(np.uint32) << np.uint32(16))",
     "return (x.astype(np.uint32) << np.uint32(15))"),
    ("decode_as_fp16", "return (x.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)",
     "return x.view(np.float16).astype(np.float64)"),
    ("decode_via_fp16_bits", "if x.dtype == np.uint16:", "if x.dtype == np.float16:"),
    ("bf16_truncate", "return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)",
     "return np.ldexp(np.trunc(np.ldexp(m, 8)), e - 8)"),
    ("bf16_fp16_width", "return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)",
     "return np.ldexp(np.rint(np.ldexp(m, 11)), e - 11)"),
    ("bf16_num_terms_unrounded", "term = bf16_round(w[r].T[:, :, None] * np.asarray(o_r, dtype=np.float64))",
     "term = w[r].T[:, :, None] * np.asarray(o_r, dtype=np.float64)"),
    ("bf16_num_final_round_only", "n = term if n is None else bf16_round(n + term)",
     "n = term if n is None else n + term"),
    ("bf16_num_unweighted", "term = bf16_round(w[r].T[:, :, None] * np.asarray(o_r, dtype=np.float64))",
     "term = bf16_round(np.asarray(o_r, dtype=np.float64))"),
    ("cyclic_block_contiguous", "pages = np.arange(shard, n_pages, n_shards, dtype=np.int64)",
     "pages = np.arange(shard * (n_pages // n_shards), (shard + 1) * (n_pages // n_shards), dtype=np.int64)"),
    ("dsa_no_relu", "out[k_] = W @ np.maximum(Q @ K.T, 0.0)", "out[k_] = W @ (Q @ K.T)"),
    ("dsa_unweighted", "out[k_] = W @ np.maximum(Q @ K.T, 0.0)", "out[k_] = np.maximum(Q @ K.T, 0.0).sum(axis=0)"),
    ("dsa_abs_not_relu", "out[k_] = W @ np.maximum(Q @ K.T, 0.0)", "out[k_] = W @ np.abs(Q @ K.T)"),
    ("topk_ties_high_pos", "order = np.lexsort((pos[r], -scores[r]))", "order = np.lexsort((-pos[r], -scores[r]))"),
    ("topk_smallest", "order = np.lexsort((pos[r], -scores[r]))", "order = np.lexsort((pos[r], scores[r]))"),
    ("topk_unsorted_out", "out[r] = np.sort(pos[r][order[:take]])", "out[r] = pos[r][order[:take]]"),
    ("key_positions_ignored", "keys = np.asarray(key_positions, dtype=np.int64)",
     "keys = np.arange(kv_begin, min(kv_end, last_visible))"),
]


def _mutant(old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor not unique/present: {old!r}"
    mod = types.ModuleType("oracle_mutant")
    exec(compile(src.replace(old, new), SRC + ":mutant", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_mutation_is_caught(name, old, new):
    mod = _mutant(old, new)
    failed = []
    for pin in ALL_PINS:
        try:
            pin(mod)
        except Exception as e:  # noqa: BLE001 - any failure counts as caught
            failed.append((pin.__name__, type(e).__name__))
    assert failed, f"mutation {name} passed every pin"
