"""fp64/bit-exact oracle of the KV refresh write -- TEST INFRASTRUCTURE ONLY.

Paper, Sec. "Infrastructure Optimization", cache control: the editing pass
reads the cache but does not write it; afterwards the blocks that changed are
recomputed under standard attention and their K/V written back, which
restores a cache consistent with standard-scope decoding.

kv_write is the write-back: token t of sequence b (absolute position
start_b + t, t < n_b) goes to slot (start_b + t) % 16 of page
page_table[b][(start_b + t) // 16], for every KV head.  The K pool is
[page][head][16][D]; the V pool [page][head][D][16] (token-minor) or, with
v_token_major, [page][head][16][D] like K.  With
block flags ([batch][blocks], block size B), token t of sequence b is
written only when flags[b][t // B] is set: the blocks the refresh recomputes.

refresh_blocks reads which blocks to recompute from the per-block changed
flags.  The paper refreshes only the changed blocks; because a later block's
standard-scope K/V attended to the old tokens, the second mode also marks
every block after the first changed one (per sequence).
"""
from __future__ import annotations

import numpy as np

PAGE = 16
REFRESH_CHANGED, REFRESH_CHANGED_AND_LATER = 0, 1


def _np(x):
    return x.detach().cpu().numpy() if hasattr(x, "detach") else np.asarray(x)


def kv_write(k_pages, v_pages, page_table, start_pos, lens, k_new, v_new, block_flags=None, block_size=None,
             v_token_major=False):
    """Returns updated copies of the two pools (same dtype as given)."""
    K = _np(k_pages).copy()
    V = _np(v_pages).copy()
    pt = _np(page_table).astype(np.int64)
    st = _np(start_pos).astype(np.int64)
    n = _np(lens).astype(np.int64)
    kn = _np(k_new)
    vn = _np(v_new)
    fl = None if block_flags is None else _np(block_flags)
    row = 0
    for b in range(st.shape[0]):
        for t in range(int(n[b])):
            if fl is None or fl[b, t // int(block_size)]:
                pos = int(st[b]) + t
                page = int(pt[b, pos // PAGE])
                slot = pos % PAGE
                K[page, :, slot, :] = kn[row]
                if v_token_major:
                    V[page, :, slot, :] = vn[row]
                else:
                    V[page, :, :, slot] = vn[row]
            row += 1
    return K, V


def refresh_blocks(block_changed, mode):
    """[batch][nblk] uint8 -> [batch][nblk] uint8 blocks to recompute."""
    C = _np(block_changed).astype(np.uint8)
    out = np.zeros_like(C)
    for b in range(C.shape[0]):
        seen = False
        for i in range(C.shape[1]):
            if C[b, i]:
                out[b, i] = 1
                seen = True
            elif seen and mode == REFRESH_CHANGED_AND_LATER:
                out[b, i] = 1
    return out
