"""Seeded random shapes through the GPU window attention, against the oracle.

Each seed draws a batch of 1..5 sequences with ragged prefixes (0..1500
tokens, any value), windows of 0..k blocks (block size 8, 16 or 32), 1, 2 or
4 KV heads with 1, 2, 4 or 8 query heads each, head_dim 64 or 128, a mask
mode, a split-KV chunk (library's choice or forced), host lengths or bounds
only, and extra unreferenced pages; every pool slot no sequence covers holds
NaN.  Together the draws reach every kernel variant: one or two waves per 64
rows (at most 128 rows per KV head), one to four query tiles per KV head,
split and unsplit, masked tails.  Odd seeds use token-major V pages.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import assert_attn_close, say

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def draw(seed):
    rng = np.random.default_rng(5000 + seed)
    batch = int(rng.integers(1, 6))
    B = int(rng.choice([8, 16, 32]))
    k = int(rng.integers(1, 5))
    Hkv = int(rng.choice([1, 2, 4]))
    G = int(rng.choice([1, 2, 4, 8]))
    D = int(rng.choice([64, 128]))
    P = [int(x) for x in rng.integers(0, 1501, size=batch)]
    W = [int(x) * B for x in rng.integers(0, k + 1, size=batch)]
    W[int(rng.integers(batch))] = k * B
    mode = str(rng.choice(["bidir", "block_causal"]))
    split = int(rng.choice([0, 0, 64, 128, 192, 512]))
    host = bool(rng.integers(2))
    extra = int(rng.integers(0, 4))
    spec = synth.AttnSpec(batch, B, k, ("fixed", 0), Hkv * G, Hkv, D)
    case = synth.make_attention_case(spec, 6000 + seed, prefix_lens=P, window_lens=W, extra_pages=extra,
                                     tail_fill=float("nan"), v_token_major=seed % 2 == 1)
    return case, mode, split, host


@pytest.mark.parametrize("seed", range(48))
def test_random_shape_parity(gpu, seed):
    case, mode, split, host = draw(seed)
    say(f"  seed {seed}: B={case.block_size} G={case.num_q_heads // case.num_kv_heads} Hkv={case.num_kv_heads} "
        f"D={case.head_dim} P={case.prefix_lens.tolist()} W={case.window_lens.tolist()} {mode} split={split} "
        f"host={host} v_token_major={case.v_token_major}")
    c = case.to(DEV)
    kw = {}
    if host:
        kw.update(host_prefix_lens=case.prefix_lens, host_window_lens=case.window_lens)
    else:
        # bounds only: looser than the true maxima
        B = case.block_size
        kw.update(max_prefix_len=int(case.prefix_lens.max()) + 7,
                  max_window_len=int(case.window_lens.max()) + B)
    out = gpu.window_attention(c.q, c.k_pages, c.v_pages, c.page_table, c.prefix_lens, c.window_lens,
                               case.block_size, mask_mode=mode, kv_split_tokens=split, **kw)
    torch.cuda.synchronize()
    m = oracle.MASK_BIDIR if mode == "bidir" else oracle.MASK_BLOCK_CAUSAL
    ref = oracle.window_attention(case.q, case.k_pages, case.v_pages, case.page_table, case.prefix_lens,
                                  case.window_lens, case.block_size, m, v_token_major=case.v_token_major)
    assert_attn_close(out.cpu(), ref, f"seed {seed}")


def test_batch_beyond_dispatch_order_table(gpu):
    """1100 short sequences: more than the 1024 whose longest-first dispatch
    order fits in the kernel arguments, so the host lengths are ignored for
    ordering and sequences run in natural order; results must not change."""
    rng = np.random.default_rng(77)
    n = 1100
    spec = synth.AttnSpec(n, 16, 2, ("fixed", 0), 2, 1, 64)
    P = [int(x) for x in rng.integers(0, 90, size=n)]
    W = [int(x) * 16 for x in rng.integers(0, 3, size=n)]
    case = synth.make_attention_case(spec, 78, prefix_lens=P, window_lens=W)
    c = case.to(DEV)
    out = gpu.window_attention(c.q, c.k_pages, c.v_pages, c.page_table, c.prefix_lens, c.window_lens, 16,
                               host_prefix_lens=case.prefix_lens, host_window_lens=case.window_lens)
    torch.cuda.synchronize()
    ref = oracle.window_attention(case.q, case.k_pages, case.v_pages, case.page_table, case.prefix_lens,
                                  case.window_lens, 16)
    assert_attn_close(out.cpu(), ref, "1100 sequences")


@pytest.mark.parametrize("mode", ["bidir", "block_causal"])
def test_many_sequences_split_merge(gpu, mode):
    """80 sequences with ragged windows and forced splits.  The main kernel and
    the split merge find a sequence's first query row by summing the window
    lengths of the sequences before it, 64 lanes at a time, so sequences past
    the 64th take a second round of that sum in both kernels."""
    rng = np.random.default_rng(91)
    n = 80
    spec = synth.AttnSpec(n, 16, 2, ("fixed", 0), 4, 2, 64)
    P = [int(x) for x in rng.integers(100, 700, size=n)]
    W = [int(x) * 16 for x in rng.integers(0, 3, size=n)]
    W[-1] = 32
    case = synth.make_attention_case(spec, 92, prefix_lens=P, window_lens=W, tail_fill=float("nan"))
    c = case.to(DEV)
    say(f"  80 sequences, {mode}, split 128")
    out = gpu.window_attention(c.q, c.k_pages, c.v_pages, c.page_table, c.prefix_lens, c.window_lens, 16,
                               mask_mode=mode, kv_split_tokens=128, host_prefix_lens=case.prefix_lens,
                               host_window_lens=case.window_lens)
    torch.cuda.synchronize()
    m = oracle.MASK_BIDIR if mode == "bidir" else oracle.MASK_BLOCK_CAUSAL
    ref = oracle.window_attention(case.q, case.k_pages, case.v_pages, case.page_table, case.prefix_lens,
                                  case.window_lens, 16, m)
    assert_attn_close(out.cpu(), ref, f"80 sequences {mode}")
