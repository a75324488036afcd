"""GPU parity of edit selection with the oracle: tokens and changed mask
bit-exact, confidence within 1e-6 relative (fp32 accumulation vs fp64)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import say

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
CONF_REL = 1e-6
AMBIGUOUS = 1e-5     # |conf - threshold| below this would make the fp32/fp64 decision unstable


@pytest.fixture(autouse=True)
def _name(request):
    say(f"\n[gpu] {request.node.nodeid}")


def run(mbe, logits, cur, thr, vocab=None):
    n, c, ch = mbe.edit_select(logits.to(DEV), cur.to(DEV), thr, vocab=vocab)
    torch.cuda.synchronize()
    return n.cpu().numpy(), c.cpu().numpy().astype(np.float64), ch.cpu().numpy()


def check(gpu_res, ref, thr, what, rows=None):
    n, c, ch = gpu_res
    rn, rc, rch = ref
    if rows is not None:
        n, c, ch = n[rows], c[rows], ch[rows]
    assert np.all(np.abs(rc - thr) >= AMBIGUOUS), f"{what}: input has rows too close to the threshold"
    bad = np.nonzero(n != rn)[0]
    assert bad.size == 0, f"{what}: new_tokens differ at rows {bad[:10]} gpu {n[bad[:5]]} ref {rn[bad[:5]]}"
    assert np.array_equal(ch, rch), f"{what}: changed mask differs"
    rel = np.max(np.abs(c - rc) / rc)
    assert rel <= CONF_REL, f"{what}: conf rel err {rel:.2e}"
    return rel


@pytest.mark.parametrize("name", ["tiny_p64_k2_h4_d64", "single_p2048_k2_gqa16x4_d128"])
def test_workload_full_parity(gpu, name):
    case = synth.workload_edit(name, cur_hit_fraction=0.25)
    res = run(gpu, case.logits, case.cur_tokens, case.threshold)
    ref = oracle.edit_select(case.logits, case.cur_tokens, case.threshold)
    rel = check(res, ref, case.threshold, name)
    say(f"  rows {case.logits.shape[0]} changed {int(res[2].sum())} conf rel err {rel:.2e}")


def test_batch32_full_parity(gpu):
    case = synth.workload_edit("batch32_p512to8192_k2", cur_hit_fraction=0.25)
    res = run(gpu, case.logits, case.cur_tokens, case.threshold)
    ref = oracle.edit_select(case.logits, case.cur_tokens, case.threshold)
    check(res, ref, case.threshold, "batch32")


def test_long_context_every_row(gpu):
    """8192 x 131072 at the benchmark size: every row against the oracle."""
    case = synth.workload_edit("long_context_b64_p4096to32768_k4", cur_hit_fraction=0.25)
    res = run(gpu, case.logits, case.cur_tokens, case.threshold)
    R = case.logits.shape[0]
    refs = []
    for r0 in range(0, R, 1024):
        sl = slice(r0, r0 + 1024)
        refs.append(oracle.edit_select(case.logits[sl], case.cur_tokens[sl], case.threshold))
        say(f"  oracle rows {r0}..{r0 + 1023}")
    ref = tuple(np.concatenate([x[i] for x in refs]) for i in range(3))
    rel = check(res, ref, case.threshold, "long_context")
    say(f"  rows {R} changed {int(res[2].sum())} conf rel err {rel:.2e}")


def test_special_rows_pin_ge_and_ties(gpu):
    V = 1024
    L = torch.zeros(6, V)
    L[1] = -5.0
    L[2, [700, 100]] = 3.0
    L[3, [5, 6, 1000]] = 7.0
    L[4] = float("-inf")
    L[4, 77] = 1.0
    L[5, 1023] = 2.0
    L = L.to(torch.bfloat16)
    cur = torch.tensor([0, 3, 700, 5, 77, 1022], dtype=torch.int32)
    n, c, ch = run(gpu, L, cur, 1.0 / V)
    assert c[0] == 1.0 / V and c[1] == 1.0 / V, c[:2]
    assert list(n) == [0, 0, 100, 5, 77, 1023] and list(ch) == [0, 1, 1, 0, 0, 1]
    assert c[4] == 1.0
    n, c, ch = run(gpu, L, cur, float(np.nextafter(np.float32(1.0 / V), np.float32(1))))
    assert list(ch[:2]) == [0, 0]
    n, c, ch = run(gpu, L, cur, 1.5)
    assert not ch.any() and np.array_equal(n, cur.numpy())
    n, c, ch = run(gpu, L, cur, 0.0)
    assert list(ch) == [0, 1, 1, 0, 0, 1]


@pytest.mark.parametrize("vocab,stride,offset", [(1000, 1000, 0), (50257, 50264, 0), (4096, 4100, 1),
                                                   (131072, 131072, 0), (7, 7, 0)])
def test_odd_vocab_strides_alignment(gpu, vocab, stride, offset):
    spec = synth.EditSpec(40, stride + offset, 3.0, 0.5, 0.5)
    case = synth.make_edit_case(spec, 13)
    full = case.logits
    view = full[:, offset:offset + stride]            # unaligned when offset is odd
    cur = torch.randint(0, vocab, (40,), dtype=torch.int32, generator=torch.Generator().manual_seed(1))
    dev_full = full.to(DEV)
    dview = dev_full[:, offset:offset + stride]
    n, c, ch = gpu.edit_select(dview, cur.to(DEV), 0.5, vocab=vocab)
    torch.cuda.synchronize()
    ref = oracle.edit_select(view[:, :vocab], cur, 0.5)
    rc = ref[1]
    keep = np.abs(rc - 0.5) >= AMBIGUOUS
    assert np.array_equal(n.cpu().numpy()[keep], ref[0][keep])
    assert np.array_equal(ch.cpu().numpy()[keep], ref[2][keep])
    assert np.max(np.abs(c.cpu().numpy() - rc) / rc) <= CONF_REL


def test_deterministic_and_chunking_invariant(gpu):
    case = synth.workload_edit("single_p2048_k2_gqa16x4_d128")     # 64 rows: split into chunks
    a = run(gpu, case.logits, case.cur_tokens, case.threshold)
    b = run(gpu, case.logits, case.cur_tokens, case.threshold)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    # same rows inside a 2048-row batch (one workgroup per row)
    big = case.logits.repeat(32, 1)
    bc = case.cur_tokens.repeat(32)
    c = run(gpu, big, bc, case.threshold)
    assert np.array_equal(c[0][:64], a[0]) and np.array_equal(c[2][:64], a[2])
    assert np.max(np.abs(c[1][:64] - a[1]) / a[1]) <= 1e-6


def test_workspace_reuse_across_row_counts(gpu):
    for rows in (64, 1000, 8, 512, 64):
        spec = synth.EditSpec(rows, 131072, 3.0, 0.5, 0.9)
        case = synth.make_edit_case(spec, rows)
        res = run(gpu, case.logits, case.cur_tokens, case.threshold)
        ref = oracle.edit_select(case.logits, case.cur_tokens, case.threshold)
        check(res, ref, case.threshold, f"rows={rows}")


def test_zero_rows(gpu):
    n, c, ch = gpu.edit_select(torch.empty(0, 128, dtype=torch.bfloat16, device=DEV),
                               torch.empty(0, dtype=torch.int32, device=DEV), 0.9)
    assert n.numel() == 0


def test_logits_beyond_2_31_elements(gpu):
    """17024 x 131072 logits (2.23e9 elements, 4.5 GB): the rows past 2^31
    elements need 64-bit row offsets.  Seeded N(0, 3) drawn on the device, a
    +8 peak in every other sampled row; 64 sampled rows, the last ones
    included, against the oracle."""
    R, V = 17024, 131072
    gen = torch.Generator(device=DEV)
    gen.manual_seed(11)
    L = torch.empty(R, V, dtype=torch.bfloat16, device=DEV).normal_(0.0, 3.0, generator=gen)
    rng = np.random.default_rng(12)
    rows = np.unique(np.concatenate([[0, R // 2, R - 2, R - 1], rng.choice(R, 60, replace=False)]))
    for r, col in zip(rows[::2], rng.integers(0, V, size=rows[::2].size)):
        L[int(r), int(col)] = (L[int(r)].float().max() + 8.0).to(torch.bfloat16)
    cur = torch.from_numpy(rng.integers(0, V, size=R).astype(np.int32))
    say(f"  {R} x {V} = {R * V:.3e} elements")
    res = run(gpu, L, cur, 0.9)
    sel = torch.from_numpy(rows)
    ref = oracle.edit_select(L[sel.to(DEV)].cpu(), cur[sel], 0.9)
    check(res, ref, 0.9, "logits beyond 2^31 elements", rows=rows)
    del L
    torch.cuda.empty_cache()
