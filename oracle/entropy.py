"""fp64 oracle of tail-entropy block selection -- TEST INFRASTRUCTURE ONLY.

Paper, Sec. "Training-Free MBE Decoding", paragraph "Tail-entropy block
selection", Eqs. (5)-(6), with the entropy H(p) = -sum_v p_v log p_v of the
model's predictive distribution at a position (the same quantity whose
exponential is the perplexity of Eq. (3)):

  S_rho(i) = mean of the ceil(rho * B) largest entropies e_{i,r} of block i
  j*       = argmax over i in C_j of S_rho(i),
             C_j = { i : max(0, j - K_max + 1) <= i < j }

Readings (where the paper is silent):
  * entropy in nats, softmax at temperature 1 over the full given vocabulary;
    -inf logits have probability 0 and contribute nothing;
  * among equal scores the earliest block wins (the widest window);
  * for j = 0, C_j is empty and the window starts at j itself.
"""
from __future__ import annotations

import math

import numpy as np


def row_entropy(logits):
    """H per row in nats, from p_v = exp(l_v - lse) as -sum p_v (l_v - lse)."""
    L = logits.detach().cpu().double().numpy() if hasattr(logits, "detach") else np.asarray(logits, np.float64)
    out = np.empty(L.shape[0], dtype=np.float64)
    for r in range(L.shape[0]):
        row = L[r]
        fin = row[np.isfinite(row)]
        mx = fin.max()
        lse = mx + math.log(np.sum(np.exp(fin - mx)))
        logp = fin - lse
        out[r] = -float(np.sum(np.exp(logp) * logp))
    return out


def tail_entropy_scores(entropy, block_size, rho):
    """S_rho(i) for every block of B consecutive rows (Eq. (5))."""
    e = np.asarray(entropy, dtype=np.float64)
    B = int(block_size)
    k = int(math.ceil(float(np.float32(rho)) * B))
    if not 1 <= k <= B:
        raise ValueError("ceil(rho * B) must lie in [1, B]")
    nblk = e.shape[0] // B
    scores = np.empty(nblk, dtype=np.float64)
    for i in range(nblk):
        top = np.sort(e[i * B:(i + 1) * B])[::-1][:k]
        scores[i] = float(np.sum(top)) / k
    return scores


def select_start_block(scores, current_block, k_max):
    """j* per sequence (Eq. (6)).  scores: [batch][max_blocks] S_rho of each
    committed block; current_block: [batch] j."""
    S = np.asarray(scores, dtype=np.float64)
    J = np.asarray(current_block, dtype=np.int64)
    out = np.empty(J.shape[0], dtype=np.int32)
    for b in range(J.shape[0]):
        j = int(J[b])
        lo = max(0, j - int(k_max) + 1)
        best = j
        for i in range(lo, j):
            if best == j or S[b, i] > S[b, best]:
                best = i
        out[b] = best
    return out
