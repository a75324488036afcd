"""GPU parity of window attention / block-diffusion attention with the oracle.

Every case calls libmbe through its C ABI (via the ctypes binding) and
compares with oracle.window_attention (fp64) on the same seeded inputs."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import assert_attn_close, say, seq_slice

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(autouse=True)
def _name(request):
    say(f"\n[gpu] {request.node.nodeid}")


def run_case(mbe, case, mode="bidir", **kw):
    c = case.to(DEV)
    out = mbe.window_attention(c.q, c.k_pages, c.v_pages, c.page_table, c.prefix_lens, c.window_lens,
                               case.block_size, mask_mode=mode, **kw)
    torch.cuda.synchronize()
    return out.cpu()


def oracle_case(case, mode="bidir"):
    m = oracle.MASK_BIDIR if mode == "bidir" else oracle.MASK_BLOCK_CAUSAL
    return oracle.window_attention(case.q, case.k_pages, case.v_pages, case.page_table,
                                   case.prefix_lens, case.window_lens, case.block_size, m,
                                   v_token_major=case.v_token_major)


# both V page layouts: token-minor [D][16] and token-major [16][D] (like K)
layouts = pytest.mark.parametrize("vt", [False, True], ids=["v_minor", "v_major"])


@layouts
@pytest.mark.parametrize("mode", ["bidir", "block_causal"])
@pytest.mark.parametrize("name", ["tiny_p64_k2_h4_d64", "single_p2048_k2_gqa16x4_d128"])
def test_workload_full_parity(gpu, name, mode, vt):
    case = synth.workload_attention(name, v_token_major=vt)
    say(f"  workload {name} mode {mode} P={case.prefix_lens.tolist()} W={case.window_lens.tolist()}")
    out = run_case(gpu, case, mode)
    err = assert_attn_close(out, oracle_case(case, mode), f"{name} {mode}")
    say(f"  max_abs {err[0]:.2e} rel_rms {err[1]:.2e}")


@layouts
@pytest.mark.parametrize("split", [64, 128, 1024])
def test_forced_split_kv(gpu, split, vt):
    case = synth.workload_attention("single_p2048_k2_gqa16x4_d128", v_token_major=vt)
    say(f"  kv_split_tokens {split}")
    out = run_case(gpu, case, "bidir", kv_split_tokens=split)
    assert_attn_close(out, oracle_case(case), f"split {split}")


@pytest.mark.parametrize("nsplit", [2, 3, 5, 8, 9, 16, 17, 32, 33, 40])
def test_merge_chunk_boundaries(gpu, nsplit):
    """Split counts on both sides of the merge's chunk sizes (8, 4, 2, 1) and
    of several chunks: a 64-key split over P + W = 64 * nsplit - 8 keys, with
    a ragged second sequence of fewer splits and one whose window is empty."""
    vt = nsplit % 2 == 1            # both V layouts over the split counts
    spec = synth.AttnSpec(3, 16, 2, ("fixed", 0), 8, 2, 64)
    P0 = 64 * nsplit - 8 - 32
    case = synth.make_attention_case(spec, 90 + nsplit, prefix_lens=[P0, max(0, P0 // 3), 100],
                                     window_lens=[32, 16, 0], tail_fill=float("nan"), v_token_major=vt)
    say(f"  nsplit {nsplit} P={case.prefix_lens.tolist()} W={case.window_lens.tolist()} v_token_major={vt}")
    for mode in ("bidir", "block_causal"):
        out = run_case(gpu, case, mode, kv_split_tokens=64)
        assert_attn_close(out, oracle_case(case, mode), f"nsplit {nsplit} {mode}")


@pytest.mark.parametrize("split", [0, 1 << 20])
def test_prefix_of_140k_keys(gpu, split):
    """A 140000-key prefix (8751 pages in its table row) beside a short one,
    with the library's split choice and with one split over the whole prefix."""
    spec = synth.AttnSpec(2, 16, 1, ("fixed", 0), 4, 2, 64)
    case = synth.make_attention_case(spec, 41, prefix_lens=[140000, 5000], window_lens=[16, 16])
    say(f"  kv_split_tokens {split} P={case.prefix_lens.tolist()}")
    for mode in ("bidir", "block_causal"):
        out = run_case(gpu, case, mode, kv_split_tokens=split, host_prefix_lens=case.prefix_lens,
                       host_window_lens=case.window_lens)
        assert_attn_close(out, oracle_case(case, mode), f"split {split} {mode}")


@layouts
@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("mode", ["bidir", "block_causal"])
def test_ragged_batch_with_poisoned_tails(gpu, D, mode, vt):
    spec = synth.AttnSpec(4, 32, 1, ("fixed", 0), 8, 2, D)
    case = synth.make_attention_case(spec, 21, prefix_lens=[0, 37, 1000, 333],
                                     window_lens=[32, 96, 64, 0], extra_pages=3,
                                     tail_fill=float("nan"), v_token_major=vt)
    say(f"  D={D} mode={mode} P={case.prefix_lens.tolist()} W={case.window_lens.tolist()}")
    for split in (0, 64, 256):
        out = run_case(gpu, case, mode, kv_split_tokens=split)
        assert_attn_close(out, oracle_case(case, mode), f"ragged D={D} {mode} split={split}")


@layouts
@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("mode", ["bidir", "block_causal"])
def test_key_split_waves_ragged(gpu, D, mode, vt):
    """At most 128 rows per (sequence, KV head) (here 2 query heads per KV head,
    windows up to 64): pairs of waves split every key tile and add their
    partial results.  Ragged prefixes, an empty window, poisoned page tails."""
    spec = synth.AttnSpec(4, 32, 1, ("fixed", 0), 8, 4, D)
    case = synth.make_attention_case(spec, 31, prefix_lens=[0, 45, 1300, 211],
                                     window_lens=[64, 32, 64, 0], extra_pages=2,
                                     tail_fill=float("nan"), v_token_major=vt)
    say(f"  D={D} mode={mode} P={case.prefix_lens.tolist()} W={case.window_lens.tolist()}")
    for split in (0, 64, 320):
        out = run_case(gpu, case, mode, kv_split_tokens=split)
        assert_attn_close(out, oracle_case(case, mode), f"key split D={D} {mode} split={split}")


@layouts
def test_key_split_waves_sharp_scores(gpu, vt):
    """Single-block windows with 16 query / 4 KV heads (128 rows: the key-split
    path) and Q scaled by 8: scores spread over tens of log2 units, so later
    keys exceed the first block's maximum (the fixed softmax reference)."""
    spec = synth.AttnSpec(3, 32, 1, ("fixed", 0), 16, 4, 128)
    case = synth.make_attention_case(spec, 41, prefix_lens=[2000, 64, 777], q_scale=8.0, v_token_major=vt)
    for split in (0, 256):
        out = run_case(gpu, case, "bidir", kv_split_tokens=split)
        assert_attn_close(out, oracle_case(case), f"key split sharp split={split}")


def _plant_hot_keys(case, seed, q_gain=6.0, hot_per_seq=5):
    """Q rows = q_gain * s + N(0,1) for one sign vector s per KV head, and a few
    keys past the first 64 of each sequence set to s * U(0.9, 1): their scores
    lie ~100 log2 units above the first 32-key block's, so the fixed-reference
    row sums overflow and the kernel must take its exact rerun."""
    rng = np.random.default_rng(seed)
    Hq, Hkv, D = case.num_q_heads, case.num_kv_heads, case.head_dim
    G = Hq // Hkv
    sgn = rng.choice([-1.0, 1.0], size=(Hkv, D))
    q = case.q.float().numpy()
    noise = rng.standard_normal(q.shape)
    q = q_gain * np.repeat(sgn, G, axis=0)[None, :, :] + noise
    k = case.k_pages.float().numpy().copy()
    pt = case.page_table.numpy()
    P, W = case.prefix_lens.numpy(), case.window_lens.numpy()
    for b in range(case.batch):
        n = int(P[b] + W[b])
        if n <= 64:
            continue
        for t in rng.choice(np.arange(64, n), size=min(hot_per_seq, n - 64), replace=False):
            page, slot = pt[b, t // 16], t % 16
            k[page, :, slot, :] = sgn * rng.uniform(0.9, 1.0, size=(Hkv, D))
    case.q = torch.from_numpy(q).to(torch.bfloat16)
    case.k_pages = torch.from_numpy(k).to(torch.bfloat16)
    return case


@layouts
@pytest.mark.parametrize("W", [32, 64])
@pytest.mark.parametrize("mode", ["bidir", "block_causal"])
def test_overflow_rerun(gpu, W, mode, vt):
    """Row sums against the first block's maximum overflow: the exact rerun
    (max-only pass, then the full pass with the true maximum) must reproduce
    the oracle.  W = 32 is the key-split path (128 rows), W = 64 the other."""
    spec = synth.AttnSpec(3, 32, W // 32, ("fixed", 0), 16, 4, 128)
    case = synth.make_attention_case(spec, 51, prefix_lens=[700, 3000, 96], v_token_major=vt)
    case = _plant_hot_keys(case, 52)
    say(f"  W={W} mode={mode} P={case.prefix_lens.tolist()}")
    for split in (0, 256):
        out = run_case(gpu, case, mode, kv_split_tokens=split)
        assert_attn_close(out, oracle_case(case, mode), f"rerun W={W} {mode} split={split}")


@pytest.mark.parametrize("B", [8, 16])
def test_small_blocks_block_causal(gpu, B):
    spec = synth.AttnSpec(2, B, 4, ("fixed", 0), 4, 4, 128)
    case = synth.make_attention_case(spec, 5, prefix_lens=[200, 13], v_token_major=B == 16)
    say(f"  block_size {B}")
    for mode in ("bidir", "block_causal"):
        out = run_case(gpu, case, mode, kv_split_tokens=128)
        assert_attn_close(out, oracle_case(case, mode), f"B={B} {mode}")


def test_sharp_scores_online_softmax(gpu):
    """Q scaled by 8: scores spread over tens of units, so the running maximum
    moves and the lazy rescale path is exercised."""
    spec = synth.AttnSpec(2, 32, 2, ("fixed", 0), 16, 4, 128)
    case = synth.make_attention_case(spec, 77, prefix_lens=[1500, 700], q_scale=8.0)
    for split in (0, 256):
        out = run_case(gpu, case, "bidir", kv_split_tokens=split)
        assert_attn_close(out, oracle_case(case), f"sharp split={split}")


@layouts
def test_block_diffusion_baseline(gpu, vt):
    spec = synth.AttnSpec(3, 32, 1, ("fixed", 0), 16, 4, 128)
    case = synth.make_attention_case(spec, 9, prefix_lens=[640, 0, 96], v_token_major=vt)
    c = case.to(DEV)
    out = gpu.block_diffusion_attention(c.q, c.k_pages, c.v_pages, c.page_table, c.prefix_lens, 32)
    torch.cuda.synchronize()
    ref = oracle.block_diffusion_attention(case.q, case.k_pages, case.v_pages, case.page_table,
                                           case.prefix_lens, 32, v_token_major=vt)
    assert_attn_close(out.cpu(), ref, "block_diffusion_attention")
    # k = 1: window bidirectional == block-causal == baseline, on the GPU path itself
    w_bi = run_case(gpu, case, "bidir")
    w_bc = run_case(gpu, case, "block_causal")
    assert torch.equal(w_bi, out.cpu()) and torch.equal(w_bc, out.cpu())


def test_block_diffusion_ragged_prefixes(gpu):
    """Ragged prefixes with host lengths: the block-diffusion call plans its
    splits from them, and its workspace comes from its own size query."""
    spec = synth.AttnSpec(5, 32, 1, ("fixed", 0), 16, 4, 128)
    case = synth.make_attention_case(spec, 19, prefix_lens=[100, 16000, 0, 3000, 544])
    c = case.to(DEV)
    out = gpu.block_diffusion_attention(c.q, c.k_pages, c.v_pages, c.page_table, c.prefix_lens, 32,
                                        host_prefix_lens=case.prefix_lens)
    torch.cuda.synchronize()
    ref = oracle.block_diffusion_attention(case.q, case.k_pages, case.v_pages, case.page_table,
                                           case.prefix_lens, 32, v_token_major=case.v_token_major)
    assert_attn_close(out.cpu(), ref, "block_diffusion_attention, ragged prefixes")


def test_block_causal_equals_stacked_single_blocks_on_gpu(gpu):
    spec = synth.AttnSpec(1, 32, 3, ("fixed", 0), 16, 4, 128)
    case = synth.make_attention_case(spec, 12, prefix_lens=[512])
    full = run_case(gpu, case, "block_causal")
    c = case.to(DEV)
    for j in range(3):
        qj = c.q[32 * j:32 * (j + 1)].contiguous()
        one = gpu.block_diffusion_attention(qj, c.k_pages, c.v_pages, c.page_table, c.prefix_lens + 32 * j, 32)
        torch.cuda.synchronize()
        a = full[32 * j:32 * (j + 1)].float()
        assert (a - one.cpu().float()).abs().max() <= 1e-2, f"block {j}"


def test_empty_inputs(gpu):
    spec = synth.AttnSpec(2, 32, 1, ("fixed", 0), 4, 4, 64)
    case = synth.make_attention_case(spec, 1, prefix_lens=[64, 16], window_lens=[0, 0])
    c = case.to(DEV)
    out = gpu.window_attention(c.q, c.k_pages, c.v_pages, c.page_table, c.prefix_lens, c.window_lens, 32)
    torch.cuda.synchronize()
    assert out.shape == (0, 4, 64)


def test_workspace_reuse_across_shapes(gpu):
    """A workspace reused by a call with more query tiles after a call whose
    partial results were larger: the counters must not have been overwritten."""
    for k, split in ((4, 0), (8, 0), (2, 1024), (8, 2048), (1, 0)):
        case = synth.workload_attention("span_sweep_b8_p16384", k_blocks=k,
                                        prefix_lens=[4096, 1000, 4000, 64, 2048, 3000, 512, 4096])
        out = run_case(gpu, case, "bidir", kv_split_tokens=split)
        for b in (1, 7):
            q, pt, P, W, rows = seq_slice(case, b)
            ref = oracle.window_attention(q, case.k_pages, case.v_pages, pt, P, W, case.block_size,
                                          v_token_major=case.v_token_major)
            assert_attn_close(out[rows], ref, f"k={k} split={split} seq {b}")


@pytest.mark.parametrize("host", [True, False])
def test_host_lengths_or_bounds_only(gpu, host):
    """With host copies of the lengths the library sizes splits from the work
    and dispatches the longest sequences first; with bounds only it uses the
    natural order.  Both must give the oracle's result."""
    spec = synth.AttnSpec(6, 32, 2, ("fixed", 0), 16, 4, 128)
    case = synth.make_attention_case(spec, 31, prefix_lens=[100, 3000, 0, 1500, 64, 2900],
                                     window_lens=[64, 32, 96, 0, 64, 32])
    c = case.to(DEV)
    kw = dict(host_prefix_lens=case.prefix_lens, host_window_lens=case.window_lens) if host else \
        dict(max_prefix_len=3000, max_window_len=96)
    for mode in ("bidir", "block_causal"):
        out = gpu.window_attention(c.q, c.k_pages, c.v_pages, c.page_table, c.prefix_lens, c.window_lens, 32,
                                   mask_mode=mode, **kw)
        torch.cuda.synchronize()
        assert_attn_close(out.cpu(), oracle_case(case, mode), f"host={host} {mode}")


def test_deterministic(gpu):
    case = synth.workload_attention("single_p2048_k2_gqa16x4_d128")
    a = run_case(gpu, case, "bidir", kv_split_tokens=256)
    b = run_case(gpu, case, "bidir", kv_split_tokens=256)
    assert torch.equal(a, b)


# ---------------------------------------------------------------- benchmark sizes, every sequence
_ORACLE_ROWS = {}     # (workload, mode, sequence) -> oracle rows; the same values in both V layouts


def _per_sequence_parity(gpu, case, seqs, what, mode="bidir", **kw):
    """One call over the whole batch at its benchmark shape (the launch the
    bench times); the oracle then runs sequence by sequence on the rows of
    `seqs` (every sequence unless a subset is given).  Both V layouts hold
    the same values, so the oracle rows of a sequence are computed once."""
    out = run_case(gpu, case, mode, **kw)
    m = oracle.MASK_BIDIR if mode == "bidir" else oracle.MASK_BLOCK_CAUSAL
    worst = (0.0, 0.0)
    for b in seqs:
        q, pt, P, W, rows = seq_slice(case, b)
        key = (what, mode, b)
        if key not in _ORACLE_ROWS:
            _ORACLE_ROWS[key] = oracle.window_attention(q, case.k_pages, case.v_pages, pt, P, W, case.block_size, m,
                                                        v_token_major=case.v_token_major)
        err = assert_attn_close(out[rows], _ORACLE_ROWS[key], f"{what} {mode} seq {b} v_token_major={case.v_token_major}")
        worst = (max(worst[0], err[0]), max(worst[1], err[1]))
        say(f"  {what} {mode} seq {b} P={int(P[0])}: max_abs {err[0]:.2e} rel_rms {err[1]:.2e}")
    say(f"  {what} {mode} v_token_major={case.v_token_major}: {len(seqs)} sequences, "
        f"worst max_abs {worst[0]:.2e} rel_rms {worst[1]:.2e}")


@layouts
def test_batch32_every_sequence(gpu, vt):
    case = synth.workload_attention("batch32_p512to8192_k2", v_token_major=vt)
    _per_sequence_parity(gpu, case, range(case.batch), "batch32")


@layouts
@pytest.mark.parametrize("k", synth.SPAN_SWEEP_K)
def test_span_sweep_every_sequence(gpu, k, vt):
    case = synth.workload_attention("span_sweep_b8_p16384", k_blocks=k, v_token_major=vt)
    _per_sequence_parity(gpu, case, range(case.batch), f"span k={k}")


@layouts
def test_long_context_every_sequence(gpu, vt):
    """All 64 sequences of the long-context workload (prefixes 4K-32K, 4-block
    windows) against the oracle."""
    case = synth.workload_attention("long_context_b64_p4096to32768_k4", v_token_major=vt)
    _per_sequence_parity(gpu, case, range(case.batch), "long_context")


@layouts
def test_long_context_block_causal_sampled(gpu, vt):
    """Block-causal (the refresh scope) at the long-context shape, 4 blocks of
    32 with prefixes up to 32K: the longest, the shortest and two other
    sequences against the oracle (the launch covers all 64)."""
    case = synth.workload_attention("long_context_b64_p4096to32768_k4", v_token_major=vt)
    P = case.prefix_lens.numpy()
    seqs = sorted({int(np.argmax(P)), int(np.argmin(P)), 9, 40})
    _per_sequence_parity(gpu, case, seqs, "long_context", mode="block_causal")


@layouts
def test_span_sweep_block_causal_k4_split(gpu, vt):
    """Block-causal with 4 blocks over a 16K prefix and forced 1024-key
    splits (the split-KV merge under the block-causal mask), every sequence."""
    case = synth.workload_attention("span_sweep_b8_p16384", k_blocks=4, v_token_major=vt)
    _per_sequence_parity(gpu, case, range(case.batch), "span k=4 split 1024", mode="block_causal",
                         kv_split_tokens=1024)


def test_debug_check_rejects_bad_device_values(gpu, monkeypatch):
    """MBE_DEBUG_CHECK=1: the attention call copies the lengths and the page
    table to the host and returns MBE_ERR_BAD_VALUE, launching nothing, for a
    page id outside the pool, a prefix beyond its bound or a window length
    that is not a multiple of the block; a valid call still matches the oracle."""
    spec = synth.AttnSpec(2, 32, 2, ("fixed", 0), 8, 2, 128)
    case = synth.make_attention_case(spec, 71, prefix_lens=[100, 300])
    c = case.to(DEV)
    monkeypatch.setenv("MBE_DEBUG_CHECK", "1")
    out = run_case(gpu, case)
    assert_attn_close(out, oracle_case(case), "debug check on, valid input")

    def call(**over):
        a = dict(page_table=c.page_table, prefix_lens=c.prefix_lens, window_lens=c.window_lens)
        kw = dict(max_prefix_len=300, max_window_len=64)
        for key in list(over):
            (a if key in a else kw)[key] = over[key]
        with pytest.raises(gpu.MbeError) as ei:
            gpu.window_attention(c.q, c.k_pages, c.v_pages, a["page_table"], a["prefix_lens"], a["window_lens"],
                                 32, **kw)
        torch.cuda.synchronize()
        return ei.value

    bad_pages = c.page_table.clone()
    bad_pages[1, 3] = case.k_pages.shape[0] + 5
    e = call(page_table=bad_pages)
    assert e.status == 6 and "page_table[1][3]" in str(e), str(e)
    neg_pages = c.page_table.clone()
    neg_pages[0, 0] = -1
    assert call(page_table=neg_pages).status == 6
    e = call(max_prefix_len=200)
    assert e.status == 6 and "prefix_lens[1]" in str(e), str(e)
    e = call(window_lens=torch.tensor([64, 48], dtype=torch.int32, device=DEV))
    assert e.status == 6 and "window_lens[1]" in str(e), str(e)


def test_two_streams_get_their_own_workspace(gpu):
    """Split-KV calls (which use the workspace) issued on two streams at once:
    each matches the oracle, so the binding's per-stream buffers do not race."""
    spec = synth.AttnSpec(1, 32, 2, ("fixed", 0), 16, 4, 128)
    a = synth.make_attention_case(spec, 91, prefix_lens=[3000])
    b = synth.make_attention_case(spec, 92, prefix_lens=[2500])
    ca, cb = a.to(DEV), b.to(DEV)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    for _ in range(3):
        with torch.cuda.stream(s1):
            oa = gpu.window_attention(ca.q, ca.k_pages, ca.v_pages, ca.page_table, ca.prefix_lens, ca.window_lens,
                                      32, kv_split_tokens=256)
        with torch.cuda.stream(s2):
            ob = gpu.window_attention(cb.q, cb.k_pages, cb.v_pages, cb.page_table, cb.prefix_lens, cb.window_lens,
                                      32, kv_split_tokens=256)
    torch.cuda.synchronize()
    assert_attn_close(oa.cpu(), oracle_case(a), "stream 1")
    assert_attn_close(ob.cpu(), oracle_case(b), "stream 2")


def test_pool_beyond_2_31_elements(gpu):
    """K/V pools of 300000 pages x 4 KV heads x 16 x 128 (2.46e9 elements,
    4.9 GB each): page ids near the end lie past 2^31 elements, so the page
    addressing of attention and of the KV write-back must be 64-bit.  One
    sequence (prefix 4000, window 64) whose pages are spread over the whole
    pool, its window on the pool's last page; the oracle runs on a compact
    copy of the referenced pages."""
    Hkv, D, Hq, B = 4, 128, 16, 32
    npages, P, W = 300_000, 4000, 64
    n_pg = (P + W + 15) // 16
    rng = np.random.default_rng(123)
    ids = rng.choice(npages - 1, size=n_pg, replace=False).astype(np.int64)
    ids[(P + W - 1) // 16] = npages - 1                   # the window's last page is the pool's last
    gen = torch.Generator(device=DEV)
    gen.manual_seed(7)
    K = torch.empty(npages, Hkv, 16, D, dtype=torch.bfloat16, device=DEV).normal_(generator=gen)
    V = torch.empty(npages, Hkv, D, 16, dtype=torch.bfloat16, device=DEV).normal_(generator=gen)
    q = torch.from_numpy(rng.normal(size=(W, Hq, D)).astype(np.float32)).to(torch.bfloat16)
    pt = torch.from_numpy(ids.astype(np.int32)[None, :])
    plen = torch.tensor([P], dtype=torch.int32)
    wlen = torch.tensor([W], dtype=torch.int32)
    say(f"  pool {npages} pages, last element offset {npages * Hkv * 16 * D:.3e}; page ids up to {ids.max()}")
    out = gpu.window_attention(q.to(DEV), K, V, pt.to(DEV), plen.to(DEV), wlen.to(DEV), B)
    torch.cuda.synchronize()
    idx = torch.from_numpy(ids).to(DEV)
    Kc, Vc = K[idx].cpu(), V[idx].cpu()
    compact = torch.arange(n_pg, dtype=torch.int32)[None, :]
    ref = oracle.window_attention(q, Kc, Vc, compact, plen, wlen, B)
    assert_attn_close(out.cpu(), ref, "attention over a pool beyond 2^31 elements")
    # KV write-back of the window tokens: lands on pages including the last
    kn = torch.from_numpy(rng.normal(size=(W, Hkv, D)).astype(np.float32)).to(torch.bfloat16)
    vn = torch.from_numpy(rng.normal(size=(W, Hkv, D)).astype(np.float32)).to(torch.bfloat16)
    gpu.kv_write(K, V, pt.to(DEV), plen.to(DEV), wlen.to(DEV), kn.to(DEV), vn.to(DEV))
    torch.cuda.synchronize()
    rk, rv = oracle.kv_write(Kc.view(torch.int16), Vc.view(torch.int16), compact.numpy(), plen.numpy(), wlen.numpy(),
                             kn.view(torch.int16), vn.view(torch.int16))
    assert np.array_equal(K[idx].cpu().view(torch.int16).numpy(), rk)
    assert np.array_equal(V[idx].cpu().view(torch.int16).numpy(), rv)
    del K, V
    torch.cuda.empty_cache()


@layouts
@pytest.mark.parametrize("mode", ["bidir", "block_causal"])
def test_dispatch_table_ragged_windows(gpu, mode, vt):
    """A small ragged batch with host lengths takes the host-placed dispatch
    table; with 8 query heads per KV head and windows of 1 to 4 blocks the
    sequences have 1 or 2 query tiles, the table's general ordering path."""
    spec = synth.AttnSpec(5, 16, 4, ("fixed", 0), 16, 2, 64)
    case = synth.make_attention_case(spec, 57, prefix_lens=[100, 3000, 700, 1500, 50],
                                     window_lens=[16, 64, 32, 48, 0], tail_fill=float("nan"), v_token_major=vt)
    out = run_case(gpu, case, mode, host_prefix_lens=case.prefix_lens, host_window_lens=case.window_lens)
    assert_attn_close(out, oracle_case(case, mode), f"dispatch table, ragged windows, {mode}")
