"""The threshold update without a workspace (mbe_threshold_update_noalloc,
through the C ABI) equals the call with a workspace bit for bit, on two
calls in a row on one GPU, the second smaller (its scratch then holds the
first call's leftovers), and on a chunked shape (rows under 512: partials in
the scratch too)."""
import numpy as np
import pytest
import torch

import synth
from gpu_util import say

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _case(name, rows, seed):
    case = synth.workload_edit(name, rows=rows)
    L, cur = case.logits, case.cur_tokens.clone()
    V = L.shape[1]
    rng = np.random.default_rng(seed)
    cur[torch.from_numpy(rng.random(rows) < 0.4)] = V - 1          # masked rows (mask id V - 1)
    return L.to(DEV), cur.to(DEV), V - 1


def _outputs(rows, block):
    return {"new_tokens": torch.full((rows,), -7, dtype=torch.int32, device=DEV),
            "conf": torch.full((rows,), -1.0, dtype=torch.float32, device=DEV),
            "action": torch.full((rows,), 9, dtype=torch.uint8, device=DEV),
            "block_changed": torch.full((rows // block,), 9, dtype=torch.uint8, device=DEV),
            "changed_count": torch.full((1,), -5, dtype=torch.int32, device=DEV),
            "entropy": torch.full((rows,), -1.0, dtype=torch.float32, device=DEV)}


def _same(a, b, what):
    for k in a:
        x, y = a[k].cpu(), b[k].cpu()
        if x.dtype == torch.float32:
            x, y = x.view(torch.int32), y.view(torch.int32)
        assert torch.equal(x, y), f"{what}: {k} differs"


def test_noalloc_matches_workspace_call_twice(gpu):
    block = 32
    for name, rows, seed in (("batch32_p512to8192_k2", 2048, 1), ("single_p2048_k2_gqa16x4_d128", 64, 2)):
        say(f"  noalloc: {name} rows {rows}")
        L, cur, mid = _case(name, rows, seed)
        ref = gpu.threshold_update(L, cur, mid, block, 0.5, 0.0, with_entropy=True, out=_outputs(rows, block))
        got = gpu.threshold_update_noalloc(L, cur, mid, block, 0.5, 0.0, out=_outputs(rows, block))
        torch.cuda.synchronize()
        _same(got, ref, f"{name} rows {rows}")
        say(f"    changed {int(got['changed_count'].item())} rows, bit-identical")
