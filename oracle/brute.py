"""Brute-force restatement of the window attention -- TEST INFRASTRUCTURE ONLY.

Independent of oracle.attention (no shared helpers): scalar Python loops,
no matrix products, and visibility taken from block ids instead of counts.

Block ids over the P + W tokens of one sequence (paper, Sec. "Block
diffusion" and Eq. (4)): committed prefix tokens carry id -1; window token u
(absolute position P + u) carries id u // B.  A window query of block c sees
  * bidirectional window mode: every token (ids -1 .. k-1);
  * block-causal (standard) mode: tokens whose id is <= c.
V pages are [page][head][D][16] (token-minor) or, with v_token_major,
[page][head][16][D].  For tiny inputs only.
"""
from __future__ import annotations

import math


def _lst(x):
    if hasattr(x, "detach"):
        x = x.detach().cpu()
        if x.is_floating_point():
            x = x.double()
        return x.tolist()
    return x.tolist() if hasattr(x, "tolist") else list(x)


def brute_window_attention(q, k_pages, v_pages, page_table, prefix_lens, window_lens,
                           block_size, bidirectional=True, softmax_scale=None, v_token_major=False):
    q, kp, vp = _lst(q), _lst(k_pages), _lst(v_pages)
    pt, P_all, W_all = _lst(page_table), _lst(prefix_lens), _lst(window_lens)
    Hq = len(q[0]) if q else 0
    D = len(q[0][0]) if q else 0
    Hkv = len(kp[0])
    page = 16
    scale = softmax_scale if softmax_scale else 1.0 / math.sqrt(D)
    out = [[[0.0] * D for _ in range(Hq)] for _ in range(len(q))]
    base = 0
    for b in range(len(P_all)):
        P, W = int(P_all[b]), int(W_all[b])
        n = P + W
        ids = [-1] * P + [u // block_size for u in range(W)]
        # visibility matrix over all (query token, key token) pairs
        visible = [[(ids[t] <= ids[s]) or bidirectional for t in range(n)] for s in range(n)]
        for u in range(W):
            s = P + u
            for h in range(Hq):
                g = h * Hkv // Hq
                scores = []
                for t in range(n):
                    if not visible[s][t]:
                        continue
                    pg, sl = pt[b][t // page], t % page
                    dot = 0.0
                    for d in range(D):
                        dot += q[base + u][h][d] * kp[pg][g][sl][d]
                    scores.append((t, dot * scale))
                mx = max(v for _, v in scores)
                w = [(t, math.exp(v - mx)) for t, v in scores]
                z = sum(e for _, e in w)
                for d in range(D):
                    acc = 0.0
                    for t, e in w:
                        pg, sl = pt[b][t // page], t % page
                        acc += e * (vp[pg][g][sl][d] if v_token_major else vp[pg][g][d][sl])
                    out[base + u][h][d] = acc / z
        base += W
    return out
