"""Shared helpers of the GPU parity tests (compare with the oracle)."""
import numpy as np
import torch

# attention tolerance: max-abs 2e-2 and relative RMS 1e-2 against the fp64 oracle
ATTN_MAX_ABS = 2e-2
ATTN_REL_RMS = 1e-2


def attn_errors(gpu_out, ref):
    g = gpu_out.detach().float().cpu().double().numpy() if hasattr(gpu_out, "detach") else np.asarray(gpu_out)
    r = np.asarray(ref, dtype=np.float64)
    assert g.shape == r.shape, (g.shape, r.shape)
    assert np.all(np.isfinite(g)), "non-finite output"
    diff = g - r
    max_abs = float(np.max(np.abs(diff))) if diff.size else 0.0
    den = float(np.linalg.norm(r))
    rel_rms = float(np.linalg.norm(diff) / den) if den > 0 else float(np.linalg.norm(diff))
    return max_abs, rel_rms


def assert_attn_close(gpu_out, ref, what):
    max_abs, rel_rms = attn_errors(gpu_out, ref)
    assert max_abs <= ATTN_MAX_ABS and rel_rms <= ATTN_REL_RMS, \
        f"{what}: max|diff| {max_abs:.3e} (tol {ATTN_MAX_ABS}), rel RMS {rel_rms:.3e} (tol {ATTN_REL_RMS})"
    return max_abs, rel_rms


def seq_slice(case, b):
    """The q rows / lengths of sequence b alone, sharing the KV pools."""
    cu = case.cu_q
    return (case.q[cu[b]:cu[b + 1]], case.page_table[b:b + 1], case.prefix_lens[b:b + 1],
            case.window_lens[b:b + 1], slice(int(cu[b]), int(cu[b + 1])))


def say(*a):
    print(*a, flush=True)
