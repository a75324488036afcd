"""Pins of the oracle's threshold update, entropy and KV-refresh functions.

Like oracle_pins.py, every check takes the oracle module under test as an
argument so that test_oracle_pin_strength.py can show that planted mistakes
are caught.

Threshold update (paper Eq. (1) and the force-unmask rule after it):
  hand-derived fixture (tests/golden/threshold_update_hand.json); the T2T part
  equals the edit-selection oracle on rows with no mask; properties on random
  blocks (every block with masks resolves at least one; Gamma rows clear
  omega_mask; the counts and flags agree with the actions).
Entropy and tail selection (Eqs. (3), (5), (6)):
  uniform over n -> ln n (perplexity n), single finite logit -> 0, two-point
  closed form (fixture); scipy.stats.entropy of scipy.special.softmax on random
  rows; invariance to a constant shift; tail scores by repeated removal of the
  maximum; start block by scanning candidates in a different order.
KV write:
  hand-derived fixture (tests/golden/kv_write_hand.json: the page and slot of
  every written row, with and without block flags, worked out by hand);
  read-back through an independent gather loop equals the written values and
  every other slot is untouched; round trip: contiguous K/V written into
  shuffled, NaN-filled pages (prefix and window in separate writes, the
  window starting mid-page) and read by the brute-force attention give the
  mean of the written V rows for q = 0 and torch's fp64 SDPA over the
  contiguous K/V for random q; refresh modes by a direct definition.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np
import scipy.special
import scipy.stats

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

_NAMED = {"ln2": math.log(2.0), "ln1.5": math.log(1.5), "ln3": math.log(3.0), "-inf": -math.inf}


def _val(s):
    return _NAMED[s] if s in _NAMED else float(s)


def _expr(s):
    e = math.e
    table = {"e^2/(e^2+3)": e ** 2 / (e ** 2 + 3), "e/(e+3)": e / (e + 3), "1/4": 0.25, "2/5": 0.4,
             "1/3": 1.0 / 3.0, "1/2": 0.5, "ln4": math.log(4.0), "ln8": math.log(8.0), "0": 0.0,
             "-(3/4)ln(3/4)-(1/4)ln(1/4)": -(0.75 * math.log(0.75)) - 0.25 * math.log(0.25)}
    return table[s]


def _fixture(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ----------------------------------------------------------------------------- update


def check_update_golden(upd):
    fx = _fixture("threshold_update_hand.json")
    L = np.array([[_val(x) for x in row] for row in fx["logits"]])
    out = upd.threshold_update(L, np.array(fx["cur"]), fx["mask_id"], fx["B"], fx["omega_mask"],
                               fx["omega_edit"])
    assert list(out["action"]) == fx["action"], (list(out["action"]), fx["action"])
    assert list(out["new_tokens"]) == fx["new_tokens"]
    assert list(out["block_changed"]) == fx["block_changed"]
    assert out["changed_count"] == fx["changed_count"]
    want = np.array([_expr(c) for c in fx["conf"]])
    assert np.allclose(out["conf"], want, rtol=1e-14, atol=0), (out["conf"], want)


def check_update_t2t_matches_edit_select(upd):
    """With no masked rows, Eq. (1) reduces to the T2T rule of the edit oracle."""
    import oracle
    rng = np.random.default_rng(11)
    R, V, B = 32, 50, 8
    L = rng.normal(0, 2, (R, V))
    cur = rng.integers(0, V - 1, R)            # mask id V - 1 never current
    L[::3, 7] += 6                             # confident rows
    cur[::6] = 7                               # some agree with the prediction
    for om, oe in ((0.5, 0.0), (0.5, 0.3), (0.9, 0.95)):
        out = upd.threshold_update(L, cur, V - 1, B, om, oe)
        new, conf, ch = oracle.edit_select(L, cur, oe)
        assert np.array_equal(out["new_tokens"], new)
        assert np.array_equal(out["action"] == 3, ch.astype(bool))
        assert np.allclose(out["conf"], conf, rtol=1e-15)


def check_update_properties(upd):
    rng = np.random.default_rng(12)
    R, V, B, mask = 64, 40, 8, 39
    for trial in range(6):
        L = rng.normal(0, 1.0 + trial, (R, V))
        cur = rng.integers(0, V - 1, R)
        cur[rng.random(R) < 0.5] = mask
        out = upd.threshold_update(L, cur, mask, B, 0.5, 0.0)
        act, new = out["action"], out["new_tokens"]
        pred = np.argmax(L, axis=1)
        conf = 1.0 / np.sum(np.exp(L - L.max(axis=1, keepdims=True)), axis=1)
        for k in range(R // B):
            rows = np.arange(k * B, (k + 1) * B)
            masked = rows[cur[rows] == mask]
            if len(masked):
                # every block with masks unmasks at least one of them
                assert np.any(act[masked] != 0)
                forced = masked[act[masked] == 2]
                assert len(forced) <= 1
                if len(forced):
                    assert not np.any(act[masked] == 1)
                    assert conf[forced[0]] == conf[masked].max()
                    assert forced[0] == masked[conf[masked] == conf[masked].max()][0]
            assert out["block_changed"][k] == int(np.any(act[rows] != 0))
        assert np.all(conf[act == 1] > 0.5)
        assert np.all(cur[act == 1] == mask) and np.all(cur[act == 3] != mask)
        assert np.all(new[act != 0] == pred[act != 0]) and np.all(new[act == 0] == cur[act == 0])
        assert out["changed_count"] == int(np.count_nonzero(act))


UPDATE_CHECKS = [check_update_golden, check_update_t2t_matches_edit_select, check_update_properties]


# ----------------------------------------------------------------------------- entropy


def check_entropy_golden(ent):
    fx = _fixture("tail_entropy_hand.json")
    for case in fx["entropy_cases"]:
        L = np.array([[_val(x) for x in case["logits"]]])
        H = ent.row_entropy(L)[0]
        assert abs(H - _expr(case["H"])) < 1e-14, (case, H)
    t = fx["tail"]
    for rho, score in t["rho_to_score"]:
        s = ent.tail_entropy_scores(np.array(t["entropy"]), t["B"], rho)
        assert abs(s[0] - score) < 1e-14, (rho, s, score)
    sel = fx["select"]
    for j, start in sel["j_to_start"]:
        got = ent.select_start_block(np.array([sel["scores"]]), np.array([j]), sel["k_max"])[0]
        assert got == start, (j, got, start)


def check_entropy_vs_scipy(ent):
    rng = np.random.default_rng(13)
    L = rng.normal(0, 3, (20, 300))
    L[3, :150] = -math.inf
    H = ent.row_entropy(L)
    for r in range(L.shape[0]):
        p = scipy.special.softmax(L[r])
        assert abs(H[r] - scipy.stats.entropy(p)) < 1e-12 * max(1.0, H[r])
    H2 = ent.row_entropy(L + 17.25)
    assert np.allclose(H, H2, rtol=1e-12, atol=1e-13)
    n = 1000
    assert abs(ent.row_entropy(np.zeros((1, n)))[0] - math.log(n)) < 1e-12   # perplexity n


def _tail_by_removal(e, B, rho):
    k = math.ceil(float(np.float32(rho)) * B)
    out = []
    for i in range(len(e) // B):
        vals = list(e[i * B:(i + 1) * B])
        tot = 0.0
        for _ in range(k):
            m = max(vals)
            tot += m
            vals.remove(m)
        out.append(tot / k)
    return np.array(out)


def check_tail_scores(ent):
    rng = np.random.default_rng(14)
    for B, rho in ((32, 0.25), (8, 0.5), (16, 1.0), (12, 0.2), (32, 0.01)):
        e = rng.gamma(2.0, 0.7, 5 * B)
        e[B:2 * B] = 1.25                      # a block of equal entropies
        s = ent.tail_entropy_scores(e, B, rho)
        assert np.allclose(s, _tail_by_removal(e, B, rho), rtol=1e-14, atol=0)


def check_select(ent):
    rng = np.random.default_rng(15)
    S = np.round(rng.random((6, 12)) * 4) / 4      # many ties
    for k_max in (2, 3, 4, 6):
        J = rng.integers(0, 12, 6)
        got = ent.select_start_block(S, J, k_max)
        for b in range(6):
            j = int(J[b])
            cands = list(range(max(0, j - k_max + 1), j))
            if not cands:
                assert got[b] == j
                continue
            best = max(S[b, i] for i in cands)
            assert got[b] == min(i for i in reversed(cands) if S[b, i] == best)


ENTROPY_CHECKS = [check_entropy_golden, check_entropy_vs_scipy, check_tail_scores, check_select]


# ----------------------------------------------------------------------------- kv write


def _kv_case(seed):
    rng = np.random.default_rng(seed)
    Hkv, D, npages = 2, 8, 12
    K = rng.normal(size=(npages, Hkv, 16, D)).astype(np.float32)
    V = rng.normal(size=(npages, Hkv, D, 16)).astype(np.float32)
    pt = np.stack([rng.permutation(npages)[:6] for _ in range(2)]).astype(np.int32)
    pt[1] = np.setdiff1d(np.arange(npages), pt[0])[:6]    # disjoint pages per sequence
    start = np.array([5, 30], dtype=np.int32)
    lens = np.array([20, 34], dtype=np.int32)
    kn = rng.normal(size=(int(lens.sum()), Hkv, D)).astype(np.float32)
    vn = rng.normal(size=(int(lens.sum()), Hkv, D)).astype(np.float32)
    return K, V, pt, start, lens, kn, vn


def check_kv_write(kv):
    K, V, pt, start, lens, kn, vn = _kv_case(16)
    K2, V2, = kv.kv_write(K, V, pt, start, lens, kn, vn)
    touched_k = np.zeros(K.shape[:3], dtype=bool)
    row = 0
    for b in range(2):
        for t in range(int(lens[b])):
            pos = int(start[b]) + t
            page = int(pt[b][pos // 16])
            for g in range(K.shape[1]):
                assert np.array_equal(K2[page, g, pos % 16], kn[row, g])
                assert np.array_equal(np.array([V2[page, g, d, pos % 16] for d in range(V.shape[2])]), vn[row, g])
                touched_k[page, g, pos % 16] = True
            row += 1
    assert np.array_equal(K2[~touched_k], K[~touched_k])
    vt = np.transpose(touched_k, (0, 1, 2))
    for page in range(K.shape[0]):
        for g in range(K.shape[1]):
            for s in range(16):
                if not vt[page, g, s]:
                    assert np.array_equal(V2[page, g, :, s], V[page, g, :, s])


def check_refresh_modes(kv):
    C = np.array([[0, 1, 0, 0], [0, 0, 0, 0], [1, 0, 1, 0], [0, 0, 0, 1]], dtype=np.uint8)
    assert np.array_equal(kv.refresh_blocks(C, 0), C)
    want = np.array([[0, 1, 1, 1], [0, 0, 0, 0], [1, 1, 1, 1], [0, 0, 0, 1]], dtype=np.uint8)
    assert np.array_equal(kv.refresh_blocks(C, 1), want)


def check_kv_write_golden(kv):
    """Every row lands on the (page, slot) the fixture gives; nothing else
    changes.  Markers: K row r of head g = (r + 1) * 10 + g in every dim, V
    row r = -(that)."""
    fx = _fixture("kv_write_hand.json")
    npg, H, D = fx["num_pages"], fx["num_kv_heads"], fx["head_dim"]
    rows = int(sum(fx["lens"]))
    kn = np.array([[[(r + 1) * 10.0 + g] * D for g in range(H)] for r in range(rows)])
    vn = -kn
    cases = [(flags, want, vt) for flags, want in ((None, fx["written_row_page_slot"]),
                                                    (fx["block_flags"], fx["written_with_flags"]))
             for vt in (False, True)]
    for flags, want, vt in cases:
        K0 = np.full((npg, H, 16, D), 0.5)
        V0 = np.full((npg, H, 16, D) if vt else (npg, H, D, 16), 0.5)
        kw = {} if flags is None else {"block_flags": np.array(flags, dtype=np.uint8),
                                        "block_size": fx["flags_block_size"]}
        K, V = kv.kv_write(K0, V0, np.array(fx["page_table"]), np.array(fx["start_pos"]), np.array(fx["lens"]),
                           kn, vn, v_token_major=vt, **kw)
        Vs = V if vt else np.swapaxes(V, 2, 3)        # [page][head][slot][D] view for the checks
        hit = np.zeros((npg, 16), dtype=bool)
        for r, page, slot in want:
            hit[page, slot] = True
            for g in range(H):
                assert np.all(K[page, g, slot, :] == kn[r, g]), (r, page, slot, K[page, g, slot])
                assert np.all(Vs[page, g, slot, :] == vn[r, g]), (r, page, slot, Vs[page, g, slot])
        for page in range(npg):
            for slot in range(16):
                if not hit[page, slot]:
                    assert np.all(K[page, :, slot, :] == 0.5) and np.all(Vs[page, :, slot, :] == 0.5), (page, slot)


def check_kv_write_round_trip(kv):
    """Contiguous K/V of two sequences written into shuffled pages filled with
    NaN, the prefix and the window in separate writes (the window starts
    mid-page), then read back by the brute-force attention: q = 0 gives the
    mean of the written V rows over the visible keys, random q gives torch's
    fp64 SDPA over the contiguous K/V (block-id mask in block-causal mode)."""
    import torch
    import oracle
    rng = np.random.default_rng(17)
    Hkv, G, D, B = 2, 2, 4, 4
    Hq = Hkv * G
    P = np.array([21, 5])
    W = np.array([8, 4])
    n = P + W
    npg = 9
    perm = rng.permutation(npg)
    need = (n + 15) // 16
    pt = np.zeros((2, 2), dtype=np.int64)
    pt[0, :need[0]] = perm[:need[0]]
    pt[1, :need[1]] = perm[need[0]:need[0] + need[1]]
    Kc = [rng.normal(size=(int(n[b]), Hkv, D)) for b in range(2)]
    Vc = [rng.normal(size=(int(n[b]), Hkv, D)) for b in range(2)]
    q = rng.normal(size=(int(W.sum()), Hq, D))
    for vt in (False, True):
        K = np.full((npg, Hkv, 16, D), np.nan)
        V = np.full((npg, Hkv, 16, D) if vt else (npg, Hkv, D, 16), np.nan)
        # prefix tokens of both sequences, then the windows from position P_b
        K, V = kv.kv_write(K, V, pt, np.zeros(2, dtype=np.int64), P,
                           np.concatenate([Kc[b][:P[b]] for b in range(2)]),
                           np.concatenate([Vc[b][:P[b]] for b in range(2)]), v_token_major=vt)
        K, V = kv.kv_write(K, V, pt, P, W, np.concatenate([Kc[b][P[b]:] for b in range(2)]),
                           np.concatenate([Vc[b][P[b]:] for b in range(2)]), v_token_major=vt)
        _round_trip_reads(oracle, K, V, pt, P, W, B, G, Hq, D, Kc, Vc, q, vt)


def _round_trip_reads(oracle, K, V, pt, P, W, B, G, Hq, D, Kc, Vc, q, vt):
    import torch
    q0 = np.zeros((int(W.sum()), Hq, D))
    out = np.array(oracle.brute_window_attention(q0, K, V, pt, P, W, B, bidirectional=True, v_token_major=vt))
    row = 0
    for b in range(2):
        for i in range(int(W[b])):
            for h in range(Hq):
                assert np.allclose(out[row + i, h], Vc[b][:, h // G].mean(axis=0), rtol=0, atol=1e-12)
        row += int(W[b])
    for bidir in (True, False):
        out = np.array(oracle.brute_window_attention(q, K, V, pt, P, W, B, bidirectional=bidir, v_token_major=vt))
        row = 0
        for b in range(2):
            ids = np.concatenate([np.full(P[b], -1), np.arange(W[b]) // B])
            allowed = torch.from_numpy(bidir | (ids[None, :] <= ids[P[b]:, None]))
            for h in range(Hq):
                qh = torch.from_numpy(q[row:row + W[b], h])[None]
                kh = torch.from_numpy(Kc[b][:, h // G])[None]
                vh = torch.from_numpy(Vc[b][:, h // G])[None]
                ref = torch.nn.functional.scaled_dot_product_attention(qh, kh, vh, attn_mask=allowed)[0].numpy()
                assert np.allclose(out[row:row + W[b], h], ref, rtol=0, atol=1e-12), (b, h, bidir)
            row += int(W[b])


KV_CHECKS = [check_kv_write_golden, check_kv_write, check_kv_write_round_trip, check_refresh_modes]
