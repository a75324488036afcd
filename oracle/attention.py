"""fp64 oracle of the MBE editing-window attention -- TEST INFRASTRUCTURE ONLY.

What is computed (paper, Sec. "Block diffusion" and Sec. "Training-Free MBE
Decoding", Eq. (4)): for sequence b the committed prefix holds P_b tokens
whose K/V sit in the paged cache; the editing window W_j covers the next
W_b = k * B tokens (k whole blocks of B tokens).  Each window query attends

  * MASK_BIDIR        -- to every prefix token and to every window token
                         (full attention within the window, Eq. (4));
  * MASK_BLOCK_CAUSAL -- to every prefix token and to window tokens of its
                         own block or earlier blocks: the standard
                         block-diffusion scope that refresh passes use.

Cached history is only read (Sec. "Infrastructure Optimization", cache
control): the window's own K/V sit in pages the caller provides.

Readings where the paper is silent: softmax scale 1/sqrt(head_dim); query
head h uses KV head h // (Hq / Hkv); no positional term inside attention.

Plain definition, not a flash algorithm: gather K/V token by token from the
page table, materialise the score matrix, softmax by the two-pass textbook
formula in fp64, multiply by V.
"""
from __future__ import annotations

import math

import numpy as np

MASK_BIDIR = 0
MASK_BLOCK_CAUSAL = 1

PAGE_SIZE = 16


def _f64(x) -> np.ndarray:
    """Exact upcast of bf16/fp32 torch tensors or numpy arrays to fp64."""
    if hasattr(x, "detach"):
        x = x.detach().cpu()
        if x.is_floating_point():
            return x.double().numpy()
        return x.numpy()
    return np.asarray(x, dtype=np.float64)


def _i64(x) -> np.ndarray:
    if hasattr(x, "detach"):
        return x.detach().cpu().numpy().astype(np.int64)
    return np.asarray(x, dtype=np.int64)


def gather_kv(k_pages, v_pages, page_table_row, n_tokens, kv_head, v_token_major=False):
    """K and V of one sequence's first n_tokens for one KV head, as [n, D].

    Token t lives in page page_table_row[t // 16] at slot t % 16.  K pages
    are [num_pages, Hkv, 16, D]; V pages are [num_pages, Hkv, D, 16]
    (token-minor) or, with v_token_major, [num_pages, Hkv, 16, D] like K.
    """
    t = np.arange(n_tokens)
    page = np.asarray(page_table_row)[t // PAGE_SIZE]
    slot = t % PAGE_SIZE
    if hasattr(k_pages, "detach"):               # torch tensor: index first, upcast after
        import torch
        page, slot = torch.from_numpy(page), torch.from_numpy(slot)
    K = _f64(k_pages[page, kv_head, slot, :])    # [n, D]
    if v_token_major:
        V = _f64(v_pages[page, kv_head, slot, :])
    else:
        V = _f64(v_pages[page, kv_head, :, slot])    # [n, D]
    return K, V


def visible_count(prefix_len, window_len, block_size, i, mask_mode):
    """Number of keys visible to window row i (keys are tokens 0..n-1)."""
    if mask_mode == MASK_BIDIR:
        return prefix_len + window_len
    if mask_mode == MASK_BLOCK_CAUSAL:
        return prefix_len + (i // block_size + 1) * block_size
    raise ValueError(f"unknown mask mode {mask_mode}")


def window_attention(q, k_pages, v_pages, page_table, prefix_lens, window_lens,
                     block_size, mask_mode=MASK_BIDIR, softmax_scale=None,
                     return_probs=False, v_token_major=False):
    """Reference output, fp64 [total_q, Hq, D].

    q [total_q, Hq, D]: rows of sequence b start at sum of earlier window
    lengths.  With return_probs, also returns {(b, h): P} where P[i, t] is the
    attention weight of window row i on key t (0 where not visible).
    """
    q = _f64(q)
    kp, vp = k_pages, v_pages                    # gathered per (sequence, head) below
    pt = _i64(page_table)
    P_all = _i64(prefix_lens)
    W_all = _i64(window_lens)
    total_q, Hq, D = q.shape
    Hkv = kp.shape[1]
    assert Hq % Hkv == 0
    G = Hq // Hkv
    scale = 1.0 / math.sqrt(D) if softmax_scale is None or softmax_scale <= 0 else float(softmax_scale)
    out = np.zeros((total_q, Hq, D))
    probs = {}
    row0 = 0
    for b in range(P_all.shape[0]):
        P, W = int(P_all[b]), int(W_all[b])
        n_all = P + W
        if W == 0:
            continue
        for g in range(Hkv):
            K, V = gather_kv(kp, vp, pt[b], n_all, g, v_token_major)
            for h in range(g * G, (g + 1) * G):
                Qb = q[row0:row0 + W, h, :]                       # [W, D]
                S = scale * (Qb @ K.T)                            # [W, n_all]
                vis = np.zeros((W, n_all), dtype=bool)
                for i in range(W):
                    vis[i, :visible_count(P, W, block_size, i, mask_mode)] = True
                S = np.where(vis, S, -np.inf)
                m = S.max(axis=1, keepdims=True)
                E = np.exp(S - m)
                Pm = E / E.sum(axis=1, keepdims=True)
                out[row0:row0 + W, h, :] = Pm @ V
                if return_probs:
                    probs[(b, h)] = Pm
        row0 += W
    if return_probs:
        return out, probs
    return out


def block_diffusion_attention(q, k_pages, v_pages, page_table, prefix_lens, block_size,
                              softmax_scale=None, v_token_major=False):
    """Standard single-block step (Sec. "Block diffusion"): block j's B queries
    see the prefix x_{0:jB} and, bidirectionally, their own block."""
    W = np.full(_i64(prefix_lens).shape[0], block_size, dtype=np.int64)
    return window_attention(q, k_pages, v_pages, page_table, prefix_lens, W, block_size,
                            MASK_BIDIR, softmax_scale, v_token_major=v_token_major)
