"""The multi-shape graph pool: every replay of a captured editing pass equals
the same calls run eagerly on the same inputs, bit for bit (same kernels, same
bounds-only plan), across several replays per shape with other GPU work and
new inputs between them, and the first replay also matches the oracle."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import assert_attn_close, say

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(autouse=True)
def _name(request):
    say(f"\n[gpu] {request.node.nodeid}")


def test_graph_pool_replays_equal_eager(gpu):
    from paper_2607_22663_amd.graphs import EditPassGraphs
    spec = synth.AttnSpec(4, 32, 2, ("fixed", 0), 16, 4, 128)
    case = synth.make_attention_case(spec, 21, prefix_lens=[96, 700, 1500, 2000])
    c = case.to(DEV)
    V, mask_id, B = 4096, 4095, 32
    max_p = 2000
    pool = EditPassGraphs(k_pages=c.k_pages, v_pages=c.v_pages, max_batch=4, max_window=64, block_size=B,
                          num_q_heads=16, max_pages_per_seq=case.page_table.shape[1], max_prefix_len=max_p,
                          vocab=V, mask_id=mask_id)
    shapes = [(4, 64), (2, 32), (4, 32)]
    for s in shapes:
        pool.capture(*s)
    rng = np.random.default_rng(22)
    for rep in range(3):
        for batch, window in shapes:
            n = batch * window
            q = torch.from_numpy(rng.normal(size=(n, 16, 128)).astype(np.float32)).to(torch.bfloat16).to(DEV)
            P = torch.from_numpy(rng.integers(0, max_p + 1, batch).astype(np.int32)).to(DEV)
            logits = torch.from_numpy(rng.normal(0, 3, (n, V)).astype(np.float32)).to(torch.bfloat16).to(DEV)
            cur = torch.from_numpy(rng.integers(0, V - 1, n).astype(np.int32))
            cur[torch.from_numpy(rng.random(n) < 0.4)] = mask_id
            cur = cur.to(DEV)
            inp = pool.inputs(batch, window)
            inp["q"].copy_(q)
            inp["page_table"].copy_(c.page_table[:batch])
            inp["prefix_lens"].copy_(P)
            inp["logits"].copy_(logits)
            inp["cur_tokens"].copy_(cur)
            pool.replay(batch, window)
            torch.cuda.synchronize()
            got = {k: v.clone() for k, v in pool.outputs(batch, window).items()}
            _ = torch.randn(1 << 20, device=DEV).sum()             # unrelated eager work between replays
            # the same calls, eagerly, on fresh tensors with the same bounds-only plan
            W = torch.full((batch,), window, dtype=torch.int32, device=DEV)
            att = gpu.window_attention(q, c.k_pages, c.v_pages, c.page_table[:batch].contiguous(), P, W, B,
                                       max_prefix_len=max_p, max_window_len=window)
            upd = gpu.threshold_update(logits, cur, mask_id, B, 0.5, 0.0, with_entropy=True)
            torch.cuda.synchronize()
            assert torch.equal(got["attention"], att), (rep, batch, window)
            for k in ("new_tokens", "conf", "action", "entropy", "block_changed", "changed_count"):
                assert torch.equal(got[k], upd[k]), (rep, batch, window, k)
            if rep == 0:
                ref = oracle.window_attention(q.cpu(), case.k_pages, case.v_pages, case.page_table[:batch],
                                              P.cpu(), W.cpu(), B)
                assert_attn_close(got["attention"], ref, f"graph replay {batch}x{window}")
                say(f"  shape {batch}x{window}: changed {int(got['changed_count'][0])}")


def test_graph_pool_rejects_unknown_shapes(gpu):
    from paper_2607_22663_amd.graphs import EditPassGraphs
    spec = synth.AttnSpec(1, 32, 1, ("fixed", 0), 4, 4, 64)
    case = synth.make_attention_case(spec, 23, prefix_lens=[64])
    c = case.to(DEV)
    pool = EditPassGraphs(k_pages=c.k_pages, v_pages=c.v_pages, max_batch=2, max_window=64, block_size=32,
                          num_q_heads=4, max_pages_per_seq=case.page_table.shape[1], max_prefix_len=64, vocab=128,
                          mask_id=127)
    with pytest.raises(ValueError):
        pool.capture(3, 32)
    with pytest.raises(ValueError):
        pool.capture(1, 48)
    with pytest.raises(KeyError):
        pool.replay(1, 32)


def test_capture_with_debug_check_enabled(gpu, monkeypatch):
    """MBE_DEBUG_CHECK=1 copies the lengths to the host, which a graph cannot
    record: calls under capture skip the check, so capture and replay still
    work, while eager calls on the same inputs are checked."""
    from paper_2607_22663_amd.graphs import EditPassGraphs
    monkeypatch.setenv("MBE_DEBUG_CHECK", "1")
    spec = synth.AttnSpec(2, 32, 1, ("fixed", 0), 4, 4, 64)
    case = synth.make_attention_case(spec, 29, prefix_lens=[64, 100])
    c = case.to(DEV)
    V, B = 256, 32
    pool = EditPassGraphs(k_pages=c.k_pages, v_pages=c.v_pages, max_batch=2, max_window=32, block_size=B,
                          num_q_heads=4, max_pages_per_seq=case.page_table.shape[1], max_prefix_len=100, vocab=V,
                          mask_id=V - 1)
    pool.capture(2, 32)
    rng = np.random.default_rng(30)
    inp = pool.inputs(2, 32)
    inp["q"].copy_(c.q)
    inp["page_table"].copy_(c.page_table)
    inp["prefix_lens"].copy_(c.prefix_lens)
    inp["logits"].copy_(torch.from_numpy(rng.normal(0, 3, (64, V)).astype(np.float32)).to(torch.bfloat16).to(DEV))
    inp["cur_tokens"].copy_(torch.from_numpy(rng.integers(0, V - 1, 64).astype(np.int32)).to(DEV))
    pool.replay(2, 32)
    torch.cuda.synchronize()
    got = pool.outputs(2, 32)["attention"].clone()
    W = torch.full((2,), 32, dtype=torch.int32, device=DEV)
    att = gpu.window_attention(c.q, c.k_pages, c.v_pages, c.page_table, c.prefix_lens, W, B,
                               max_prefix_len=100, max_window_len=32)
    torch.cuda.synchronize()
    assert torch.equal(got, att)
