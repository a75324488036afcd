"""CPU oracle for the MBE editing-pass hot path -- TEST INFRASTRUCTURE ONLY.

Plain, slow, fp64 numpy implementations of what the GPU library computes,
written from the paper (Beyond Block Boundaries: Multi-Block Editing for
Diffusion Large Language Models):

  attention.window_attention   Sec. "Training-Free MBE Decoding", Eq. (4):
                               window queries attend to the committed prefix
                               and to every window token; block-causal scope
                               of Sec. "Block diffusion" for refresh/standard
                               forwards.
  brute.brute_window_attention independent scalar-loop restatement of the
                               same visibility rule, for tiny inputs.
  edit_select.edit_select      Sec. "Configurable threshold decoding",
                               Eq. (1), the token-to-token (T2T) set Delta_t.
  update.threshold_update      Eq. (1) in full: mask-to-token set Gamma_t,
                               force-unmask, T2T set Delta_t, per-block flags.
  entropy.row_entropy, tail_entropy_scores, select_start_block
                               Sec. "Training-Free MBE Decoding", tail-entropy
                               block selection, Eqs. (5)-(6).
  kv_cache.kv_write, refresh_blocks
                               Sec. "Infrastructure Optimization", cache
                               control: write-back of recomputed K/V.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may
import this package.  It shares no code with the HIP path and never imports
it; the product path must not call it.
"""
from .attention import window_attention, block_diffusion_attention, MASK_BIDIR, MASK_BLOCK_CAUSAL
from .brute import brute_window_attention
from .edit_select import edit_select
from .entropy import row_entropy, tail_entropy_scores, select_start_block
from .kv_cache import kv_write, refresh_blocks
from .update import threshold_update

__all__ = ["window_attention", "block_diffusion_attention", "brute_window_attention",
           "edit_select", "MASK_BIDIR", "MASK_BLOCK_CAUSAL", "threshold_update", "row_entropy",
           "tail_entropy_scores", "select_start_block", "kv_write", "refresh_blocks"]
