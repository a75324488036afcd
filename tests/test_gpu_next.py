"""GPU parity of the threshold update, entropy, tail-entropy selection, KV
write-back and refresh flags with the oracle.

Bars: predictions, actions, new tokens, block flags, changed counts, start
blocks, refresh flags and the written pools are bit-exact; confidences within
1e-6 relative; entropies within 1e-4 + 2e-5 H nats (fp32 sums of 2^y and
2^y y over up to 131072 terms against fp64); tail scores within 1e-6 relative
(fp32 sum of at most B values).  The decisions compare fp32 confidences with
thresholds on the GPU and fp64 ones in the oracle, so every input is checked
to keep each confidence at least 1e-5 away from omega_mask and omega_edit, and
masked rows of one block either bitwise equal (an exact tie) or 1e-5 apart.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import say

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
CONF_REL = 1e-6
MARGIN = 1e-5


@pytest.fixture(autouse=True)
def _name(request):
    say(f"\n[gpu] {request.node.nodeid}")


def update_case(name, seed, *, block=32, mask_frac=0.4, rows=None, ties=True):
    """An edit-selection workload with masked rows (mask id V - 1) and, per
    block, one masked row copied onto another (an exact confidence tie)."""
    case = synth.workload_edit(name, rows=rows) if rows else synth.workload_edit(name)
    L = case.logits
    R, V = L.shape
    R = R // block * block
    L = L[:R].clone()
    cur = case.cur_tokens[:R].clone()
    rng = np.random.default_rng(seed)
    masked = rng.random(R) < mask_frac
    cur[torch.from_numpy(masked)] = V - 1
    if ties:
        for k in range(R // block):
            m = np.nonzero(masked[k * block:(k + 1) * block])[0]
            if len(m) >= 2:
                L[k * block + m[-1]] = L[k * block + m[0]]
    return L, cur, V - 1


def safe(L64_conf, cur, mask_id, block, om, oe):
    """Checks that no confidence lies within MARGIN of a threshold, and
    returns the blocks whose force-unmask choice fp32 cannot decide: no
    masked row clears omega_mask and the two highest masked confidences
    differ by less than MARGIN relative (without being equal).  There any
    masked row within MARGIN of the maximum is a correct choice."""
    c = np.asarray(L64_conf)
    assert np.all(np.abs(c - om) >= MARGIN) and np.all(np.abs(c - oe) >= MARGIN), "confidence too close to a threshold"
    curn = cur.numpy()
    ambiguous = []
    for k in range(len(c) // block):
        cm = np.sort(c[k * block:(k + 1) * block][curn[k * block:(k + 1) * block] == mask_id])
        if len(cm) >= 2 and cm[-1] <= om and 0 < cm[-1] - cm[-2] < MARGIN * cm[-1]:
            ambiguous.append(k)
    return ambiguous


def run_update(mbe, L, cur, mask_id, block, om, oe, entropy=True):
    out = mbe.threshold_update(L.to(DEV), cur.to(DEV), mask_id, block, om, oe, with_entropy=entropy)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def compare_update(got, ref, what, rows=None, block_ids=None, ambiguous=(), cur=None, mask_id=None, block=None):
    """Bit-exact actions and tokens, except in `ambiguous` blocks (see safe),
    where the GPU's force-unmask row only has to be a valid choice."""
    sl = slice(None) if rows is None else rows
    skip = np.zeros(len(ref["action"]), dtype=bool)
    for k in ambiguous:
        r = np.arange(k * block, (k + 1) * block)
        ga, ra = got["action"][sl][r], ref["action"][r]
        forced = r[ga == 2]
        assert len(forced) == 1, f"{what}: block {k} has {len(forced)} force-unmasked rows"
        cm = ref["conf"][r][cur[r] == mask_id]
        f = forced[0]
        assert cur[f] == mask_id and ref["conf"][f] >= cm.max() * (1 - MARGIN), f"{what}: invalid force-unmask row {f}"
        others = (ra != 2) & (ga != 2)
        assert np.array_equal(ga[others], ra[others]), f"{what}: block {k} differs beyond the force-unmask choice"
        assert np.array_equal(got["new_tokens"][sl][r][others], ref["new_tokens"][r][others])
        skip[r] = True
    for key in ("new_tokens", "action"):
        g = got[key][sl]
        bad = np.nonzero((g != ref[key]) & ~skip)[0]
        assert bad.size == 0, f"{what}: {key} differs at rows {bad[:8]}: gpu {g[bad[:5]]} ref {ref[key][bad[:5]]}"
    bc = got["block_changed"] if block_ids is None else got["block_changed"][block_ids]
    assert np.array_equal(bc, ref["block_changed"]), f"{what}: block_changed differs"
    rel = np.max(np.abs(got["conf"][sl] - ref["conf"]) / ref["conf"])
    assert rel <= CONF_REL, f"{what}: conf rel err {rel:.2e}"
    if "entropy" in ref:
        h, rh = got["entropy"][sl].astype(np.float64), ref["entropy"]
        err = np.abs(h - rh) - (1e-4 + 2e-5 * rh)
        assert np.all(err <= 0), f"{what}: entropy off by {np.max(np.abs(h - rh)):.2e} at row {np.argmax(err)}"
    return rel


@pytest.mark.parametrize("name,block,oe", [("tiny_p64_k2_h4_d64", 32, 0.0), ("tiny_p64_k2_h4_d64", 16, 0.3),
                                           ("single_p2048_k2_gqa16x4_d128", 32, 0.0),
                                           ("single_p2048_k2_gqa16x4_d128", 8, 0.95)])
def test_update_full_parity(gpu, name, block, oe):
    """Whole workloads; 64 rows x 131072 also runs the chunked path."""
    L, cur, mid = update_case(name, 1, block=block)
    ref = oracle.threshold_update(L, cur, mid, block, 0.5, oe, with_entropy=True)
    amb = safe(ref["conf"], cur, mid, block, 0.5, oe)
    got = run_update(gpu, L, cur, mid, block, 0.5, oe)
    rel = compare_update(got, ref, name, ambiguous=amb, cur=cur.numpy(), mask_id=mid, block=block)
    assert int(got["changed_count"][0]) == ref["changed_count"]
    say(f"  rows {L.shape[0]} actions {np.bincount(got['action'], minlength=4)} conf rel {rel:.1e}")


def test_update_entropy_with_neg_inf_logits(gpu):
    """64 x 131072 rows (vector loads, rows split over several workgroups) in
    which a third of the vocabulary of the first 16 rows, and all but five
    entries of row 3, are -inf: the entropy pass that meets a -inf logit goes
    through its clamped second pass and must still match the oracle, and the
    untouched rows must not change."""
    L, cur, mid = update_case("single_p2048_k2_gqa16x4_d128", 6)
    rng = np.random.default_rng(8)
    V = L.shape[1]
    Lm = L.clone()
    for r in range(16):
        Lm[r, torch.from_numpy(rng.choice(V - 1, V // 3, replace=False))] = float("-inf")
    keep = rng.choice(V - 1, 5, replace=False)
    row3 = torch.full((V,), float("-inf"), dtype=L.dtype)
    row3[torch.from_numpy(keep)] = Lm[3, torch.from_numpy(keep)]
    row3[torch.from_numpy(keep[:1])] = 4.0      # a clear maximum among the five
    Lm[3] = row3
    ref = oracle.threshold_update(Lm, cur, mid, 32, 0.5, 0.0, with_entropy=True)
    safe(ref["conf"], cur, mid, 32, 0.5, 0.0)
    got = run_update(gpu, Lm, cur, mid, 32, 0.5, 0.0)
    compare_update(got, ref, "-inf logits")
    assert np.all(np.isfinite(got["entropy"]))
    plain = run_update(gpu, L, cur, mid, 32, 0.5, 0.0)
    for key in ("conf", "entropy", "new_tokens"):
        assert np.array_equal(got[key][16:], plain[key][16:]), key


def test_update_long_context_every_block(gpu):
    """8192 x 131072 at the benchmark size: all 256 blocks against the oracle
    (run 32 blocks at a time; blocks are independent)."""
    L, cur, mid = update_case("long_context_b64_p4096to32768_k4", 2)
    B = 32
    got = run_update(gpu, L, cur, mid, B, 0.5, 0.0)
    parts = []
    for r0 in range(0, L.shape[0], 32 * B):
        sl = slice(r0, r0 + 32 * B)
        parts.append(oracle.threshold_update(L[sl], cur[sl], mid, B, 0.5, 0.0, with_entropy=True))
        say(f"  oracle rows {r0}..{r0 + 32 * B - 1}")
    ref = {k: np.concatenate([p[k] for p in parts]) for k in ("new_tokens", "conf", "action", "block_changed",
                                                               "entropy")}
    ref["changed_count"] = sum(p["changed_count"] for p in parts)
    amb = safe(ref["conf"], cur, mid, B, 0.5, 0.0)
    rel = compare_update(got, ref, "long-context, every block", ambiguous=amb, cur=cur.numpy(), mask_id=mid, block=B)
    say(f"  blocks whose force-unmask fp32 cannot decide: {amb}")
    assert int(got["changed_count"][0]) == ref["changed_count"]
    say(f"  blocks {L.shape[0] // B} actions {np.bincount(got['action'], minlength=4)} conf rel {rel:.1e}")


def test_update_exact_cases(gpu):
    """The hand-derived fixture (vocabulary 4, scalar loads, exact ties and a
    confidence exactly at omega_mask) through the GPU."""
    import json
    import os
    fx = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "threshold_update_hand.json")))
    named = {"ln2": math.log(2), "ln1.5": math.log(1.5), "-inf": -math.inf}
    L = torch.tensor([[named.get(x, None) if x in named else float(x) for x in r] for r in fx["logits"]],
                     dtype=torch.float64)
    Lb = L.to(torch.bfloat16)
    # the fixture's exact reasoning needs these logits to survive bf16: only the
    # exact-tie and exact-1/2 rows matter for the rule; compare against the
    # oracle on the bf16 values
    cur = torch.tensor(fx["cur"], dtype=torch.int32)
    got = run_update(gpu, Lb, cur, fx["mask_id"], fx["B"], fx["omega_mask"], fx["omega_edit"])
    ref = oracle.threshold_update(Lb, cur, fx["mask_id"], fx["B"], fx["omega_mask"], fx["omega_edit"],
                                  with_entropy=True)
    assert list(ref["action"]) == fx["action"]          # bf16 rounding keeps every decision of the fixture
    compare_update(got, ref, "fixture")
    assert int(got["changed_count"][0]) == fx["changed_count"]


def test_update_count_resets_between_calls(gpu):
    L, cur, mid = update_case("tiny_p64_k2_h4_d64", 4)
    a = run_update(gpu, L, cur, mid, 32, 0.5, 0.0)
    b = run_update(gpu, L, cur, mid, 32, 0.5, 0.0)
    assert int(a["changed_count"][0]) == int(b["changed_count"][0]) == int(np.count_nonzero(a["action"]))
    for k in a:
        assert np.array_equal(a[k], b[k]), k        # deterministic, including conf and entropy bits


def test_update_without_optional_outputs(gpu):
    L, cur, mid = update_case("tiny_p64_k2_h4_d64", 5)
    dev = {"new_tokens": torch.empty(64, dtype=torch.int32, device=DEV),
           "conf": torch.empty(64, dtype=torch.float32, device=DEV),
           "action": torch.empty(64, dtype=torch.uint8, device=DEV),
           "block_changed": torch.empty(2, dtype=torch.uint8, device=DEV)}
    gpu.threshold_update(L.to(DEV), cur.to(DEV), mid, 32, 0.5, 0.0, out=dev)
    full = run_update(gpu, L, cur, mid, 32, 0.5, 0.0)
    for k in dev:
        assert np.array_equal(dev[k].cpu().numpy(), full[k]), k


def test_edit_select_unchanged_by_update_mode(gpu):
    """The T2T-only call still matches the update on rows without masks."""
    case = synth.workload_edit("tiny_p64_k2_h4_d64")
    n, c, ch = gpu.edit_select(case.logits.to(DEV), case.cur_tokens.to(DEV), 0.3)
    got = run_update(gpu, case.logits, case.cur_tokens, case.logits.shape[1] + 5, 32, 0.5, 0.3)
    assert np.array_equal(n.cpu().numpy(), got["new_tokens"])
    assert np.array_equal(c.cpu().numpy(), got["conf"])
    assert np.array_equal(ch.cpu().numpy(), (got["action"] == 3).astype(np.uint8))


@pytest.mark.parametrize("B,rho", [(32, 0.25), (32, 1.0), (8, 0.5), (12, 0.2), (1024, 0.25), (5, 0.01)])
def test_tail_entropy_scores(gpu, B, rho):
    rng = np.random.default_rng(B)
    nblk = 300
    e = rng.gamma(2.0, 0.7, nblk * B).astype(np.float32)
    e[:B] = 1.5                                            # a block of equal values
    e[B:2 * B] = np.round(e[B:2 * B] * 4) / 4              # many ties
    got = gpu.tail_entropy_scores(torch.from_numpy(e).to(DEV), B, rho).cpu().numpy()
    ref = oracle.tail_entropy_scores(e.astype(np.float64), B, rho)
    assert np.max(np.abs(got - ref) / ref) <= 1e-6


def test_select_start_block(gpu):
    rng = np.random.default_rng(7)
    S = (np.round(rng.random((300, 40)) * 4) / 4).astype(np.float32)
    for k_max in (1, 2, 4, 7):
        J = rng.integers(0, 41, 300).astype(np.int32)
        J[:3] = (0, 1, 40)
        got = gpu.select_start_block(torch.from_numpy(S).to(DEV), torch.from_numpy(J).to(DEV), k_max).cpu().numpy()
        ref = oracle.select_start_block(S.astype(np.float64), J, k_max)
        assert np.array_equal(got, ref), (k_max, np.nonzero(got != ref)[0][:5])


@pytest.mark.parametrize("mode", ["changed", "changed_and_later"])
def test_refresh_blocks(gpu, mode):
    rng = np.random.default_rng(8)
    C = (rng.random((500, 9)) < 0.15).astype(np.uint8)
    got = gpu.refresh_blocks(torch.from_numpy(C).to(DEV), mode).cpu().numpy()
    ref = oracle.refresh_blocks(C, {"changed": 0, "changed_and_later": 1}[mode])
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("D,Hkv", [(128, 4), (64, 2)])
def test_kv_write(gpu, D, Hkv):
    rng = np.random.default_rng(D)
    batch, npages, maxp = 5, 200, 30
    K = torch.from_numpy(rng.normal(size=(npages, Hkv, 16, D)).astype(np.float32)).to(torch.bfloat16)
    V = torch.from_numpy(rng.normal(size=(npages, Hkv, D, 16)).astype(np.float32)).to(torch.bfloat16)
    perm = rng.permutation(npages)[: batch * maxp].reshape(batch, maxp).astype(np.int32)
    start = np.array([0, 5, 31, 64, 300], dtype=np.int32)        # aligned, mid-page, page end, later
    lens = np.array([32, 27, 1, 96, 64], dtype=np.int32)
    T = int(lens.sum())
    kn = torch.from_numpy(rng.normal(size=(T, Hkv, D)).astype(np.float32)).to(torch.bfloat16)
    vn = torch.from_numpy(rng.normal(size=(T, Hkv, D)).astype(np.float32)).to(torch.bfloat16)
    Kd, Vd = K.to(DEV), V.to(DEV)
    gpu.kv_write(Kd, Vd, torch.from_numpy(perm).to(DEV), torch.from_numpy(start).to(DEV),
                 torch.from_numpy(lens).to(DEV), kn.to(DEV), vn.to(DEV))
    rk, rv = oracle.kv_write(K.view(torch.int16), V.view(torch.int16), perm, start, lens, kn.view(torch.int16),
                             vn.view(torch.int16))
    assert np.array_equal(Kd.cpu().view(torch.int16).numpy(), rk)
    assert np.array_equal(Vd.cpu().view(torch.int16).numpy(), rv)


def test_kv_write_then_attention_reads_it(gpu):
    """A refresh written with kv_write is what the next attention call reads:
    attention over the rewritten pools equals the oracle on them."""
    case = synth.workload_attention("tiny_p64_k2_h4_d64")
    P, W = int(case.prefix_lens[0]), int(case.window_lens[0])
    rng = np.random.default_rng(9)
    T = W
    kn = torch.from_numpy(rng.normal(size=(T, case.num_kv_heads, case.head_dim)).astype(np.float32)).to(torch.bfloat16)
    vn = torch.from_numpy(rng.normal(size=(T, case.num_kv_heads, case.head_dim)).astype(np.float32)).to(torch.bfloat16)
    c = case.to(DEV)
    gpu.kv_write(c.k_pages, c.v_pages, c.page_table, torch.tensor([P], dtype=torch.int32, device=DEV),
                 torch.tensor([T], dtype=torch.int32, device=DEV), kn.to(DEV), vn.to(DEV))
    out = gpu.window_attention(c.q, c.k_pages, c.v_pages, c.page_table, c.prefix_lens, c.window_lens,
                               case.block_size)
    torch.cuda.synchronize()
    ref = oracle.window_attention(case.q, c.k_pages.cpu(), c.v_pages.cpu(), case.page_table, case.prefix_lens,
                                  case.window_lens, case.block_size)
    from gpu_util import assert_attn_close
    assert_attn_close(out, ref, "attention after kv_write")
