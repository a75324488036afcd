"""fp64 oracle of confidence-based edit selection -- TEST INFRASTRUCTURE ONLY.

Paper, Sec. "Configurable threshold decoding", Eq. (1): at position i the
prediction x_hat_i is the highest-probability token and its confidence c_i is
that probability under the model's softmax; a visible token is overwritten
(T2T set Delta_t) when x_hat_i differs from the current token and c_i clears
the edit threshold.  MBE keeps this acceptance rule for its cross-block
passes (Sec. "Training-Free MBE Decoding").

Readings where the paper is silent or differs from the library contract:
  * ties in the maximum go to the lowest vocabulary index;
  * the threshold test is c_i >= threshold (Eq. (1) writes a strict >; at the
    paper's omega_edit = 0 both agree, since c_i >= 1/V > 0);
  * softmax at temperature 1 over the full given vocabulary;
  * the threshold arrives as an fp32 value and is compared in fp64.
"""
from __future__ import annotations

import numpy as np


def edit_select(logits, cur_tokens, threshold):
    """Returns (new_tokens int32 [R], conf float64 [R], changed uint8 [R])."""
    if hasattr(logits, "detach"):
        L = logits.detach().cpu().double().numpy()
    else:
        L = np.asarray(logits, dtype=np.float64)
    cur = np.asarray(cur_tokens.cpu().numpy() if hasattr(cur_tokens, "cpu") else cur_tokens,
                     dtype=np.int64)
    R = L.shape[0]
    theta = float(np.float32(threshold))
    new = np.empty(R, dtype=np.int32)
    conf = np.empty(R, dtype=np.float64)
    changed = np.empty(R, dtype=np.uint8)
    for r in range(R):
        row = L[r]
        a = int(np.argmax(row))                 # first index of the maximum
        c = 1.0 / np.sum(np.exp(row - row[a]))  # softmax probability of a
        ch = (a != cur[r]) and (c >= theta)
        new[r] = a if ch else cur[r]
        conf[r] = c
        changed[r] = 1 if ch else 0
    return new, conf, changed
