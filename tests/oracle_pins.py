"""Checks that pin the CPU oracle to facts other than itself.

Every check takes the oracle implementation as an argument, so that
test_oracle_pin_strength.py can run the same checks against copies of the
oracle with a planted mistake and show that each mistake is caught.

Attention pins (paper, Sec. "Block diffusion" and Eq. (4)):
  brute force on tiny inputs, independent code (block ids, scalar loops);
  k = 1: bidirectional == block-causal == torch fp64 SDPA over prefix+block;
  block-causal over k blocks == k single-block steps with growing prefixes;
  prefix 0 and the window covering the whole sequence == dense SDPA;
  rows of the softmax sum to one and vanish outside the visible keys;
  invariance to a consistent page permutation, GQA == MHA with repeated KV
  heads, invariance to a consistent permutation of prefix keys (bidirectional);
  closed forms: V constant -> output is that constant; q = 0 -> mean of V;
  hand-derived fixtures in tests/golden; a token-major V pool against SDPA
  over a plain-loop gather of the same values.
Edit-selection pins (Eq. (1)):
  first-occurrence argmax by a scalar loop; confidence == max of
  scipy.special.softmax; constant rows -> (0, 1/V); ties -> lower index;
  planted peaks found; threshold semantics (>=, > 1, 0); golden fixture.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np
import torch
import torch.nn.functional as F

import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# ----------------------------------------------------------------------------------------
# helpers that do not use the oracle
# ----------------------------------------------------------------------------------------

def small_case(seed, *, batch=2, B=8, k=2, Hq=4, Hkv=2, D=16, prefix=(24, 40),
               q_scale=1.0, window_lens=None):
    spec = synth.AttnSpec(batch, B, k, ("fixed", 0), Hq, Hkv, D)
    return synth.make_attention_case(spec, seed, prefix_lens=list(prefix)[:batch],
                                     window_lens=window_lens, q_scale=q_scale)


def loop_gather(case, b, g, n):
    """K and V of sequence b, KV head g, tokens 0..n-1, fp64 torch, by a plain loop."""
    D = case.head_dim
    K = torch.empty(n, D, dtype=torch.float64)
    V = torch.empty(n, D, dtype=torch.float64)
    for t in range(n):
        page = int(case.page_table[b, t // 16])
        K[t] = case.k_pages[page, g, t % 16, :].double()
        V[t] = case.v_pages[page, g, :, t % 16].double()
    return K, V


def q_rows(case, b):
    cu = case.cu_q
    return case.q[cu[b]:cu[b + 1]].double()       # [W, Hq, D]


def sdpa(qm, K, V, mask=None):
    """torch fp64 scaled_dot_product_attention for one head: qm [W, D], K/V [n, D]."""
    return F.scaled_dot_product_attention(qm[None], K[None], V[None], attn_mask=mask)[0]


def assert_close(a, b, tol, what):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, f"{what}: shape {a.shape} vs {b.shape}"
    err = np.max(np.abs(a - b)) if a.size else 0.0
    assert err <= tol, f"{what}: max |diff| {err:.3e} > {tol:.1e}"


# ----------------------------------------------------------------------------------------
# attention pins
# ----------------------------------------------------------------------------------------

def check_brute_force(impl, brute):
    for seed, (batch, B, k, Hq, Hkv, D, prefix) in enumerate([
            (1, 4, 2, 2, 1, 8, (0,)),
            (2, 4, 3, 2, 2, 4, (5, 17)),        # prefix not a multiple of B
            (1, 8, 1, 3, 1, 8, (16,)),
            (2, 2, 2, 4, 2, 4, (1, 30)),
    ]):
        case = small_case(seed + 100, batch=batch, B=B, k=k, Hq=Hq, Hkv=Hkv, D=D, prefix=prefix)
        for mode, bidir in ((impl.MASK_BIDIR, True), (impl.MASK_BLOCK_CAUSAL, False)):
            o = impl.window_attention(case.q, case.k_pages, case.v_pages, case.page_table,
                                      case.prefix_lens, case.window_lens, B, mode)
            r = brute(case.q, case.k_pages, case.v_pages, case.page_table, case.prefix_lens,
                      case.window_lens, B, bidirectional=bidir)
            assert_close(o, r, 1e-12, f"brute force, seed {seed}, bidir={bidir}")


def check_k1_is_block_diffusion(impl):
    case = small_case(7, k=1, Hq=4, Hkv=4, D=16, prefix=(32, 9))
    B = case.block_size
    a = impl.window_attention(case.q, case.k_pages, case.v_pages, case.page_table,
                              case.prefix_lens, case.window_lens, B, impl.MASK_BIDIR)
    c = impl.window_attention(case.q, case.k_pages, case.v_pages, case.page_table,
                              case.prefix_lens, case.window_lens, B, impl.MASK_BLOCK_CAUSAL)
    d = impl.block_diffusion_attention(case.q, case.k_pages, case.v_pages, case.page_table,
                                       case.prefix_lens, B)
    assert_close(a, c, 1e-13, "k=1 bidirectional vs block-causal")
    assert_close(a, d, 1e-13, "k=1 window vs block_diffusion_attention")
    cu = case.cu_q
    for b in range(case.batch):
        n = int(case.prefix_lens[b]) + B
        for h in range(case.num_q_heads):
            g = h // (case.num_q_heads // case.num_kv_heads)
            K, V = loop_gather(case, b, g, n)
            ref = sdpa(q_rows(case, b)[:, h], K, V)
            assert_close(a[cu[b]:cu[b + 1], h], ref.numpy(), 1e-12, f"k=1 vs SDPA b={b} h={h}")


def check_block_causal_is_stacked_blocks(impl):
    """Block-causal over k blocks == k single-block steps, step j with prefix P + j*B."""
    k = 3
    case = small_case(11, batch=2, B=8, k=k, prefix=(16, 7))
    B = case.block_size
    full = impl.window_attention(case.q, case.k_pages, case.v_pages, case.page_table,
                                 case.prefix_lens, case.window_lens, B, impl.MASK_BLOCK_CAUSAL)
    cu = case.cu_q
    for b in range(case.batch):
        for j in range(k):
            rows = slice(cu[b] + j * B, cu[b] + (j + 1) * B)
            one = impl.block_diffusion_attention(
                case.q[rows], case.k_pages, case.v_pages, case.page_table[b:b + 1],
                case.prefix_lens[b:b + 1] + j * B, B)
            assert_close(full[rows], one, 1e-13, f"block-causal block {j} of seq {b}")


def check_full_window_is_dense(impl):
    case = small_case(13, batch=1, B=8, k=4, Hq=2, Hkv=1, D=16, prefix=(0,))
    B = case.block_size
    o = impl.window_attention(case.q, case.k_pages, case.v_pages, case.page_table,
                              case.prefix_lens, case.window_lens, B, impl.MASK_BIDIR)
    n = int(case.window_lens[0])
    K, V = loop_gather(case, 0, 0, n)
    for h in range(2):
        assert_close(o[:, h], sdpa(q_rows(case, 0)[:, h], K, V).numpy(), 1e-12,
                     f"dense bidirectional h={h}")
    # block-causal with prefix 0 == SDPA with a block-lower-triangular mask
    oc = impl.window_attention(case.q, case.k_pages, case.v_pages, case.page_table,
                               case.prefix_lens, case.window_lens, B, impl.MASK_BLOCK_CAUSAL)
    blk = torch.arange(n) // B
    mask = blk[None, :] <= blk[:, None]
    for h in range(2):
        assert_close(oc[:, h], sdpa(q_rows(case, 0)[:, h], K, V, mask).numpy(), 1e-12,
                     f"dense block-causal h={h}")


def check_prefix_and_window_is_sdpa(impl):
    """P > 0 and k > 1 against torch's fp64 SDPA over the gathered P + W keys:
    bidirectional = no mask at all (every window row sees the whole prefix and
    window, Eq. (4)); block-causal = the prefix plus window blocks up to the
    row's own, an explicit boolean mask built from block ids."""
    case = small_case(29, batch=2, B=8, k=3, Hq=4, Hkv=2, D=16, prefix=(21, 40))
    B = case.block_size
    ob = impl.window_attention(case.q, case.k_pages, case.v_pages, case.page_table,
                               case.prefix_lens, case.window_lens, B, impl.MASK_BIDIR)
    oc = impl.window_attention(case.q, case.k_pages, case.v_pages, case.page_table,
                               case.prefix_lens, case.window_lens, B, impl.MASK_BLOCK_CAUSAL)
    cu = case.cu_q
    G = case.num_q_heads // case.num_kv_heads
    for b in range(case.batch):
        P, W = int(case.prefix_lens[b]), int(case.window_lens[b])
        key_blk = torch.cat([torch.full((P,), -1), torch.arange(W) // B])     # prefix keys: block -1
        row_blk = torch.arange(W) // B
        mask = key_blk[None, :] <= row_blk[:, None]
        for h in range(case.num_q_heads):
            K, V = loop_gather(case, b, h // G, P + W)
            qm = q_rows(case, b)[:, h]
            assert_close(ob[cu[b]:cu[b + 1], h], sdpa(qm, K, V).numpy(), 1e-12, f"bidir vs SDPA b={b} h={h}")
            assert_close(oc[cu[b]:cu[b + 1], h], sdpa(qm, K, V, mask).numpy(), 1e-12,
                         f"block-causal vs SDPA b={b} h={h}")


def check_probs_normalised(impl):
    case = small_case(17, batch=2, B=4, k=3, prefix=(12, 3), q_scale=4.0)
    for mode in (impl.MASK_BIDIR, impl.MASK_BLOCK_CAUSAL):
        _, probs = impl.window_attention(case.q, case.k_pages, case.v_pages, case.page_table,
                                         case.prefix_lens, case.window_lens, case.block_size,
                                         mode, return_probs=True)
        for (b, h), Pm in probs.items():
            assert_close(Pm.sum(axis=1), np.ones(Pm.shape[0]), 1e-12, "row sums")
            P_b = int(case.prefix_lens[b])
            for i in range(Pm.shape[0]):
                n_i = Pm.shape[1] if mode == impl.MASK_BIDIR else P_b + (i // case.block_size + 1) * case.block_size
                assert np.all(Pm[i, n_i:] == 0.0), "weight on an invisible key"
                assert np.all(Pm[i, :n_i] > 0.0), "visible key with zero weight"


def _permute_pages(case, seed):
    rng = np.random.default_rng(seed)
    n = case.k_pages.shape[0]
    perm = rng.permutation(n)                      # new slot of old page p is perm[p]
    inv = np.argsort(perm)
    k2 = case.k_pages[torch.from_numpy(inv)]
    v2 = case.v_pages[torch.from_numpy(inv)]
    pt2 = torch.from_numpy(perm.astype(np.int32))[case.page_table.long()]
    return k2, v2, pt2


def check_invariances(impl):
    case = small_case(19, batch=2, B=8, k=2, Hq=4, Hkv=2, D=16, prefix=(40, 21))
    B = case.block_size
    args = (case.prefix_lens, case.window_lens, B)
    for mode in (impl.MASK_BIDIR, impl.MASK_BLOCK_CAUSAL):
        base = impl.window_attention(case.q, case.k_pages, case.v_pages, case.page_table, *args, mode)
        # consistent page permutation
        k2, v2, pt2 = _permute_pages(case, 5)
        o = impl.window_attention(case.q, k2, v2, pt2, *args, mode)
        assert_close(o, base, 1e-13, "page permutation")
        # GQA == MHA with KV heads repeated
        G = case.num_q_heads // case.num_kv_heads
        kr = case.k_pages.repeat_interleave(G, dim=1)
        vr = case.v_pages.repeat_interleave(G, dim=1)
        o = impl.window_attention(case.q, kr, vr, case.page_table, *args, mode)
        assert_close(o, base, 1e-13, "GQA vs repeated-KV MHA")
    # bidirectional: permuting prefix tokens consistently in K and V changes nothing
    base = impl.window_attention(case.q, case.k_pages, case.v_pages, case.page_table, *args,
                                 impl.MASK_BIDIR)
    rng = np.random.default_rng(3)
    k3, v3 = case.k_pages.clone(), case.v_pages.clone()
    for b in range(case.batch):
        P = int(case.prefix_lens[b])
        perm = rng.permutation(P)
        for t, s in enumerate(perm):
            pt, ps = int(case.page_table[b, t // 16]), t % 16
            qt, qs = int(case.page_table[b, s // 16]), s % 16
            k3[pt, :, ps, :] = case.k_pages[qt, :, qs, :]
            v3[pt, :, :, ps] = case.v_pages[qt, :, :, qs]
    o = impl.window_attention(case.q, k3, v3, case.page_table, *args, impl.MASK_BIDIR)
    assert_close(o, base, 1e-12, "prefix key permutation (bidirectional)")


def check_closed_forms(impl):
    case = small_case(23, batch=2, B=8, k=2, prefix=(33, 0))
    B = case.block_size
    args = (case.page_table, case.prefix_lens, case.window_lens, B)
    # V constant per KV head -> output equals that constant
    v = torch.empty_like(case.v_pages)
    consts = [0.5, -2.0]
    for g in range(case.num_kv_heads):
        v[:, g] = consts[g]
    G = case.num_q_heads // case.num_kv_heads
    for mode in (impl.MASK_BIDIR, impl.MASK_BLOCK_CAUSAL):
        o = impl.window_attention(case.q, case.k_pages, v, *args, mode)
        for h in range(case.num_q_heads):
            assert_close(o[:, h], np.full(o[:, h].shape, consts[h // G]), 1e-13, "constant V")
    # q = 0 -> uniform weights -> mean of the visible V rows
    q0 = torch.zeros_like(case.q)
    for mode in (impl.MASK_BIDIR, impl.MASK_BLOCK_CAUSAL):
        o = impl.window_attention(q0, case.k_pages, case.v_pages, *args, mode)
        cu = case.cu_q
        for b in range(case.batch):
            P, W = int(case.prefix_lens[b]), int(case.window_lens[b])
            for h in range(case.num_q_heads):
                _, V = loop_gather(case, b, h // G, P + W)
                for i in range(W):
                    n_i = P + W if mode == impl.MASK_BIDIR else P + (i // B + 1) * B
                    assert_close(o[cu[b] + i, h], V[:n_i].mean(0).numpy(), 1e-13, "q=0 mean")


def _golden_attention_inputs(fx):
    """Build the fixture's tensors.  Keys/values are listed per token."""
    D = fx["head_dim"]
    n = len(fx["key_first_coord_log_weights"])
    pool_pages = fx["pool_pages"]
    k_pages = np.zeros((pool_pages, 1, 16, D))
    v_pages = np.zeros((pool_pages, 1, D, 16))
    table = fx["page_table"]
    for t in range(n):
        page = table[0][t // 16]
        k_pages[page, 0, t % 16, 0] = math.log(fx["key_first_coord_log_weights"][t])
        v_pages[page, 0, t, t % 16] = 1.0           # V row t = one-hot(t)
    q = np.zeros((fx["window_len"], 1, D))
    q[:, 0, 0] = 1.0
    return q, k_pages, v_pages, np.array(table), np.array([fx["prefix_len"]]), np.array([fx["window_len"]])


def _frac(s):
    a, b = s.split("/")
    return float(a) / float(b)


def check_golden_attention(impl):
    with open(os.path.join(GOLDEN, "attention_closed_form.json")) as f:
        fx = json.load(f)
    q, kp, vp, pt, P, W = _golden_attention_inputs(fx)
    for mode_name, mode in (("bidirectional", impl.MASK_BIDIR), ("block_causal", impl.MASK_BLOCK_CAUSAL)):
        o = impl.window_attention(q, kp, vp, pt, P, W, fx["block_size"], mode, softmax_scale=1.0)
        want = np.array([[_frac(s) for s in row] for row in fx["expected"][mode_name]])
        assert_close(o[:, 0, :want.shape[1]], want, 1e-14, f"golden attention {mode_name}")


def check_token_major_v(impl):
    """A token-major V pool ([page][head][16][D]: the token-minor pool
    transposed per page) gives torch fp64 SDPA over the keys and values that a
    plain loop gathers from the token-minor pool.  head_dim 16 makes both pool
    shapes equal, so reading one layout as the other gives wrong values
    instead of a shape error."""
    case = small_case(31, k=2, Hq=4, Hkv=2, D=16, prefix=(24, 7))
    vt = case.v_pages.transpose(2, 3).contiguous()
    G = case.num_q_heads // case.num_kv_heads
    for mode in (impl.MASK_BIDIR, impl.MASK_BLOCK_CAUSAL):
        o = impl.window_attention(case.q, case.k_pages, vt, case.page_table, case.prefix_lens, case.window_lens,
                                  case.block_size, mode, v_token_major=True)
        cu = case.cu_q
        for b in range(case.batch):
            P, W = int(case.prefix_lens[b]), int(case.window_lens[b])
            ids = torch.cat([torch.full((P,), -1), torch.arange(W) // case.block_size])
            mask = (ids[None, :] <= ids[P:, None]) | (mode == impl.MASK_BIDIR)
            for h in range(case.num_q_heads):
                K, V = loop_gather(case, b, h // G, P + W)
                ref = sdpa(q_rows(case, b)[:, h], K, V, mask)
                assert_close(o[cu[b]:cu[b + 1], h], ref.numpy(), 1e-12, f"token-major V, seq {b} head {h}")


ATTENTION_CHECKS = [check_token_major_v, check_k1_is_block_diffusion, check_block_causal_is_stacked_blocks,
                    check_full_window_is_dense, check_prefix_and_window_is_sdpa, check_probs_normalised,
                    check_invariances,
                    check_closed_forms, check_golden_attention]


# ----------------------------------------------------------------------------------------
# edit-selection pins
# ----------------------------------------------------------------------------------------

def first_max_loop(row):
    best, idx = -math.inf, -1
    for v, x in enumerate(row):
        if x > best:
            best, idx = x, v
    return idx


def check_edit_argmax_conf(impl):
    import scipy.special
    spec = synth.EditSpec(48, 1024, 2.0, 0.5, 0.9)
    case = synth.make_edit_case(spec, 31)
    new, conf, changed = impl.edit_select(case.logits, case.cur_tokens, case.threshold)
    L = case.logits.double().numpy()
    sm = scipy.special.softmax(L, axis=1)
    cur = case.cur_tokens.numpy()
    for r in range(L.shape[0]):
        a = first_max_loop(L[r].tolist())
        assert abs(conf[r] - sm[r].max()) <= 1e-14, "conf vs scipy softmax"
        assert abs(conf[r] - sm[r, a]) <= 1e-14, "conf is the probability of the argmax"
        ch = (a != cur[r]) and conf[r] >= 0.9
        assert changed[r] == ch, f"changed row {r}"
        assert new[r] == (a if ch else cur[r]), f"new token row {r}"
    for r, c in zip(case.planted_rows, case.planted_cols):
        assert new[r] == c or (cur[r] == c), "planted peak not selected"
        assert changed[r] == (cur[r] != c)


def check_edit_special_rows(impl):
    V = 1024
    L = np.zeros((6, V))
    L[1] = -5.0
    L[2, [700, 100]] = 3.0                      # tie: lower index 100 wins
    L[3, [5, 6, 1000]] = [7.0, 7.0, 7.0]        # three-way tie
    L[4] = -np.inf
    L[4, 77] = 1.0                              # single finite entry
    L[5, 1023] = 2.0
    cur = np.array([0, 3, 700, 5, 77, 1022], dtype=np.int32)
    new, conf, changed = impl.edit_select(L.astype(np.float32), cur, 1.0 / V)
    assert conf[0] == 1.0 / V and conf[1] == 1.0 / V, "constant row confidence"
    assert list(new[:2]) == [0, 0] and list(changed[:2]) == [0, 1], "constant rows pin >= at 1/V"
    assert new[2] == 100 and changed[2] == 1, "tie goes to lower index"
    assert new[3] == 5 and changed[3] == 0, "three-way tie, current token already argmax"
    assert conf[4] == 1.0 and new[4] == 77 and changed[4] == 0, "single finite entry"
    assert new[5] == 1023 and changed[5] == 1
    # threshold above one: nothing changes; threshold zero: change iff argmax differs
    new, conf, changed = impl.edit_select(L.astype(np.float32), cur, 1.5)
    assert not changed.any() and np.array_equal(new, cur)
    new, conf, changed = impl.edit_select(L.astype(np.float32), cur, 0.0)
    assert list(changed) == [0, 1, 1, 0, 0, 1]
    # the same constant rows just above 1/V do not change
    new, conf, changed = impl.edit_select(L[:2].astype(np.float32), cur[:2],
                                          float(np.nextafter(np.float32(1.0 / V), np.float32(1))))
    assert not changed.any()


def check_golden_edit(impl):
    with open(os.path.join(GOLDEN, "edit_select_closed_form.json")) as f:
        fx = json.load(f)
    for c in fx["cases"]:
        row = np.array([[math.log(w) if w > 0 else -math.inf for w in c["softmax_weights"]]])
        new, conf, changed = impl.edit_select(row, np.array([c["cur"]], np.int32), c["threshold"])
        assert abs(conf[0] - _frac(c["conf"])) <= 1e-15, f"golden conf {c['name']}"
        assert int(new[0]) == c["new"] and int(changed[0]) == c["changed"], f"golden {c['name']}"


EDIT_CHECKS = [check_edit_argmax_conf, check_edit_special_rows, check_golden_edit]
