"""fp64 oracle of the full threshold update -- TEST INFRASTRUCTURE ONLY.

Paper, Sec. "Configurable threshold decoding", Eq. (1), and the paragraph after
it.  At step t every position i has a prediction x_hat_i (highest-probability
token) with confidence c_i (its probability).  With M_t the masked positions:

  Gamma_t = { i in M_t     : c_i > omega_mask }               mask-to-token
  Delta_t = { i not in M_t : x_hat_i != x_i, c_i > omega_edit } token-to-token

Positions in Gamma_t take x_hat_i, positions in Delta_t are overwritten by
x_hat_i; both use the same forward prediction.  When Gamma_t is empty while
masks remain, the masked position with the highest confidence is unmasked
(force-unmask), so a block resolves in at most B steps.

Readings (where the paper is silent):
  * M_t, Gamma_t and the force-unmask are per block of B consecutive rows (a
    block is the unit of denoising, Sec. "Block diffusion");
  * a position is masked when its current token equals the mask token id;
  * Gamma_t uses the strict test of Eq. (1); Delta_t uses the library's edit
    rule c_i >= omega_edit (identical at the paper's omega_edit = 0);
  * force-unmask ties go to the lowest row; argmax ties to the lowest token;
  * thresholds arrive as fp32 values and are compared in fp64.

Action codes per row: 0 keep, 1 unmask (Gamma), 2 force-unmask, 3 edit (Delta).
"""
from __future__ import annotations

import numpy as np

from .entropy import row_entropy

KEEP, UNMASK, FORCE_UNMASK, EDIT = 0, 1, 2, 3


def _as_f64(x):
    if hasattr(x, "detach"):
        return x.detach().cpu().double().numpy()
    return np.asarray(x, dtype=np.float64)


def _as_i64(x):
    if hasattr(x, "cpu"):
        x = x.cpu().numpy()
    return np.asarray(x, dtype=np.int64)


def prediction(logits):
    """(x_hat, c) per row: first index of the row maximum and its softmax
    probability, c = 1 / sum_v exp(l_v - l_max)."""
    L = _as_f64(logits)
    pred = np.argmax(L, axis=1)
    mx = L[np.arange(L.shape[0]), pred]
    conf = 1.0 / np.sum(np.exp(L - mx[:, None]), axis=1)
    return pred.astype(np.int64), conf


def threshold_update(logits, cur_tokens, mask_id, block_size, omega_mask, omega_edit, with_entropy=False):
    """Returns a dict with new_tokens int32 [R], conf float64 [R], action
    uint8 [R], block_changed uint8 [R / B], changed_count int and, when asked,
    entropy float64 [R] (nats)."""
    L = _as_f64(logits)
    cur = _as_i64(cur_tokens)
    R = L.shape[0]
    B = int(block_size)
    if B < 1 or R % B != 0:
        raise ValueError("rows must be a whole number of blocks")
    om = float(np.float32(omega_mask))
    oe = float(np.float32(omega_edit))
    pred, conf = prediction(L)
    masked = cur == int(mask_id)
    new = cur.copy()
    action = np.zeros(R, dtype=np.uint8)
    for r in range(R):
        if masked[r]:
            if conf[r] > om:
                action[r] = UNMASK
        elif pred[r] != cur[r] and conf[r] >= oe:
            action[r] = EDIT
    nblk = R // B
    for k in range(nblk):
        rows = range(k * B, (k + 1) * B)
        m_rows = [r for r in rows if masked[r]]
        if m_rows and not any(action[r] == UNMASK for r in m_rows):
            best = m_rows[0]
            for r in m_rows[1:]:
                if conf[r] > conf[best]:
                    best = r
            action[best] = FORCE_UNMASK
    for r in range(R):
        if action[r] != KEEP:
            new[r] = pred[r]
    block_changed = np.array([1 if np.any(action[k * B:(k + 1) * B] != KEEP) else 0 for k in range(nblk)],
                             dtype=np.uint8)
    out = {"new_tokens": new.astype(np.int32), "conf": conf, "action": action,
           "block_changed": block_changed, "changed_count": int(np.count_nonzero(action))}
    if with_entropy:
        out["entropy"] = row_entropy(L)
    return out
