"""Seeded random shapes through edit selection and the full threshold update,
against the oracle.

Each seed draws the rows (1..300), a vocabulary (1 to 200003, odd sizes
included), a row stride of vocab .. vocab + 37, a start offset of 0..7
elements (unaligned rows take the scalar-load path), logits N(0, sigma) with
sigma in {0.5, 2, 3, 8}, rows whose maximum is tied in two or three columns,
rows with -inf entries, planted peaks, and current tokens that sometimes are
the argmax.  Thresholds come from a fixed list, skipping those that some
row's confidence lies within 1e-5 of (the fp32/fp64 decision is not stable
there).  Edit selection: tokens and changed mask bit-exact, confidence within
1e-6 relative.  The update takes whole blocks of 8, 16 or 32 rows with 40% of
the rows masked (mask id V - 1)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import say
from test_gpu_next import MARGIN, compare_update, run_update

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
VOCABS = [1, 2, 7, 1000, 1024, 4099, 32000, 65536, 131072, 151936, 200003]


def draw(seed):
    rng = np.random.default_rng(9000 + seed)
    block = int(rng.choice([8, 16, 32]))
    rows = block * int(rng.integers(1, 300 // block + 1))
    V = int(rng.choice(VOCABS))
    stride = V + int(rng.integers(0, 38))
    off = int(rng.integers(0, 8))
    sigma = float(rng.choice([0.5, 2.0, 3.0, 8.0]))
    L = rng.normal(0.0, sigma, size=(rows, stride)).astype(np.float32)
    Lb = torch.from_numpy(L).to(torch.bfloat16).float().numpy()     # the values the kernels see
    for r in range(rows):
        u = rng.random()
        if u < 0.3 and V >= 3:            # tied maximum
            cols = rng.choice(V, size=int(rng.integers(2, 4)), replace=False)
            Lb[r, cols] = Lb[r, :V].max()
        elif u < 0.6:                     # planted peak
            Lb[r, int(rng.integers(V))] = Lb[r, :V].max() + float(rng.uniform(2.0, 10.0))
        if rng.random() < 0.2 and V >= 4:  # some -inf entries (never the whole row)
            Lb[r, rng.choice(V, size=max(1, V // 8), replace=False)] = -np.inf
            if np.all(np.isneginf(Lb[r, :V])):
                Lb[r, 0] = 0.0
    full = torch.empty(off + rows * stride, dtype=torch.bfloat16)
    full[off:] = torch.from_numpy(Lb.reshape(-1)).to(torch.bfloat16)
    logits = full[off:].view(rows, stride)
    first = np.argmax(Lb[:, :V], axis=1).astype(np.int32)
    cur = rng.integers(0, V, size=rows).astype(np.int32)
    hit = rng.random(rows) < 0.25
    cur[hit] = first[hit]
    return full, off, rows, stride, V, block, torch.from_numpy(cur)


def pick(conf, cands):
    for t in cands:
        if np.all(np.abs(conf - t) >= MARGIN):
            return t
    return None


@pytest.mark.parametrize("seed", range(32))
def test_random_edit_select_and_update(gpu, seed):
    full, off, rows, stride, V, block, cur = draw(seed)
    say(f"  seed {seed}: rows {rows} vocab {V} stride {stride} offset {off} block {block}")
    fd = full.to(DEV)
    Ld = fd[off:].view(rows, stride)                 # data pointer off * 2 bytes past an aligned one
    Lh = full[off:].view(rows, stride)[:, :V].contiguous()
    ref_n, ref_c, ref_ch = oracle.edit_select(Lh, cur, 1.0)
    thr = pick(ref_c, [0.9, 0.5, 0.25, 0.99, 0.0, 1.5])
    assert thr is not None
    ref_n, ref_c, ref_ch = oracle.edit_select(Lh, cur, thr)
    n, c, ch = gpu.edit_select(Ld, cur.to(DEV), thr, vocab=V)
    torch.cuda.synchronize()
    n, c, ch = n.cpu().numpy(), c.cpu().numpy().astype(np.float64), ch.cpu().numpy()
    assert np.array_equal(n, ref_n), f"tokens differ at rows {np.nonzero(n != ref_n)[0][:8]}"
    assert np.array_equal(ch, ref_ch), "changed mask differs"
    assert np.max(np.abs(c - ref_c) / ref_c) <= 1e-6
    # full update on the same rows (aligned copy), when no confidence is ambiguous
    if V < 2:
        return
    cu = cur.clone()
    cu[torch.from_numpy(np.random.default_rng(seed).random(rows) < 0.4)] = V - 1
    om = pick(ref_c, [0.5, 0.3, 0.7, 0.05])
    oe = pick(ref_c, [0.0, 0.9, 0.6])
    cm = np.sort(ref_c)
    if om is None or oe is None:
        say("  update skipped: no unambiguous thresholds")
        return
    ref = oracle.threshold_update(Lh, cu, V - 1, block, om, oe, with_entropy=True)
    # masked confidences of one block tie exactly or lie apart (force-unmask order)
    for k in range(rows // block):
        sel = cu[k * block:(k + 1) * block].numpy() == V - 1
        cmb = np.sort(ref["conf"][k * block:(k + 1) * block][sel])
        gaps = np.diff(cmb)
        if not np.all((gaps == 0) | (gaps >= MARGIN * cmb[1:])):
            say("  update skipped: masked confidences too close")
            return
    got = run_update(gpu, Lh, cu, V - 1, block, om, oe)
    compare_update(got, ref, f"seed {seed} update")
    assert int(got["changed_count"][0]) == ref["changed_count"]
