"""Seeded generator checks (CPU only)."""
import numpy as np
import torch

import synth


def test_deterministic_per_seed():
    spec = synth.WORKLOADS["tiny_p64_k2_h4_d64"].attn
    a = synth.make_attention_case(spec, 0)
    b = synth.make_attention_case(spec, 0)
    c = synth.make_attention_case(spec, 1)
    assert torch.equal(a.q, b.q) and torch.equal(a.k_pages, b.k_pages) and torch.equal(a.page_table, b.page_table)
    assert not torch.equal(a.q, c.q)


def test_page_table_is_a_permutation_of_the_pool():
    spec = synth.AttnSpec(5, 32, 2, ("uniform32", 1, 20), 4, 2, 64)
    case = synth.make_attention_case(spec, 9)
    P = case.prefix_lens.numpy()
    W = case.window_lens.numpy()
    assert np.all(P % 32 == 0) and np.all((P >= 32) & (P <= 640))
    assert np.all(W == 64)
    used = []
    for b in range(5):
        n = (int(P[b]) + int(W[b]) + 15) // 16
        used.extend(case.page_table[b, :n].tolist())
    assert sorted(used) == list(range(case.k_pages.shape[0]))
    assert case.k_pages.shape == (case.k_pages.shape[0], 2, 16, 64)
    assert case.v_pages.shape == (case.k_pages.shape[0], 2, 64, 16)
    assert case.q.dtype == torch.bfloat16 and case.q.shape == (int(W.sum()), 4, 64)


def test_tail_fill_marks_only_unreferenced_slots():
    spec = synth.AttnSpec(2, 8, 1, ("fixed", 0), 2, 1, 16)
    case = synth.make_attention_case(spec, 3, prefix_lens=[5, 20], extra_pages=2, tail_fill=float("nan"))
    nan_k = torch.isnan(case.k_pages[:, 0, :, 0])
    n_ref = 0
    for b, n in enumerate([13, 28]):
        for t in range(n):
            assert not nan_k[case.page_table[b, t // 16], t % 16]
            n_ref += 1
    assert int(nan_k.sum()) == case.k_pages.shape[0] * 16 - n_ref


def test_planted_peaks_and_cur_hits():
    spec = synth.EditSpec(40, 4096, 3.0, 0.5, 0.9)
    case = synth.make_edit_case(spec, 5, cur_hit_fraction=0.5)
    L = case.logits.float()
    assert len(case.planted_rows) == 20
    for r, c in zip(case.planted_rows, case.planted_cols):
        row = L[r]
        assert row[c] == row.max() and (row[c] - torch.topk(row, 2).values[1]) >= 7.5
    hits = sum(int(case.cur_tokens[r]) == int(c) for r, c in zip(case.planted_rows, case.planted_cols))
    assert hits == 10


def test_workload_shapes():
    w = synth.WORKLOADS["long_context_b64_p4096to32768_k4"]
    rng = synth._rng(w.seed, 0)
    P = synth.draw_prefix_lens(rng, w.attn)
    assert P.shape == (64,) and P.min() >= 4096 and P.max() <= 32768 and np.all(P % 32 == 0)
    assert w.edit.rows == 8192 and w.edit.vocab == 131072
