"""Both key loops of the attention on every kind of shape.

With token-minor V pages and no key split the library runs the
software-pipelined key loop when a work unit spans at least 96 key tiles and
the plain loop otherwise; MBE_ATTN_PIPELINE=1 / 0 forces one or the other.
Here the pipelined loop runs on the random shapes (token-minor seeds), the
overflow rerun, sharp scores, poisoned ragged tails and forced splits, and
the plain loop on the workloads that take the pipelined one by default
(long-context; spans of 8 blocks); also block flags, the device gate and
the overflow rerun at head_dim 64 through the pipelined loop; all against
the oracle.
"""
import pytest

import synth
import test_gpu_attention as A
import test_gpu_attention_random as R
import test_gpu_refresh_loop as RL
from gpu_util import assert_attn_close

pytestmark = pytest.mark.gpu


@pytest.fixture
def pipelined(monkeypatch):
    monkeypatch.setenv("MBE_ATTN_PIPELINE", "1")


@pytest.fixture
def plain(monkeypatch):
    monkeypatch.setenv("MBE_ATTN_PIPELINE", "0")


@pytest.mark.parametrize("seed", range(0, 48, 2))       # even seeds: token-minor V
def test_random_shape_parity_pipelined(gpu, pipelined, seed):
    R.test_random_shape_parity(gpu, seed)


@pytest.mark.parametrize("W", [32, 64])
@pytest.mark.parametrize("mode", ["bidir", "block_causal"])
def test_overflow_rerun_pipelined(gpu, pipelined, W, mode):
    A.test_overflow_rerun(gpu, W, mode, False)


def test_sharp_scores_pipelined(gpu, pipelined):
    A.test_sharp_scores_online_softmax(gpu)


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("mode", ["bidir", "block_causal"])
def test_ragged_batch_with_poisoned_tails_pipelined(gpu, pipelined, D, mode):
    A.test_ragged_batch_with_poisoned_tails(gpu, D, mode, False)


@pytest.mark.parametrize("split", [64, 128, 1024])
def test_forced_split_kv_pipelined(gpu, pipelined, split):
    A.test_forced_split_kv(gpu, split, False)


@pytest.mark.parametrize("name", ["tiny_p64_k2_h4_d64", "single_p2048_k2_gqa16x4_d128"])
@pytest.mark.parametrize("mode", ["bidir", "block_causal"])
def test_workload_full_parity_pipelined(gpu, pipelined, name, mode):
    A.test_workload_full_parity(gpu, name, mode, False)


def test_long_context_every_sequence_plain(gpu, plain):
    A.test_long_context_every_sequence(gpu, False)


def test_span_k8_every_sequence_plain(gpu, plain):
    A.test_span_sweep_every_sequence(gpu, 8, False)


@pytest.mark.parametrize("k", [2, 4])
def test_span_every_sequence_pipelined(gpu, pipelined, k):
    A.test_span_sweep_every_sequence(gpu, k, False)


@pytest.mark.parametrize("mode", ["bidir", "block_causal"])
def test_attention_block_flags_pipelined(gpu, pipelined, mode):
    """Block flags (targeted refresh): the pipelined kernels' workgroup OR
    goes through LDS words of their fifth tile buffer, which workgroups with
    no flagged row take before leaving.  (Split 0: that test's split runs
    use token-major V, which has no pipelined loop.)"""
    RL.test_attention_block_flags(gpu, mode, 0)


@pytest.mark.parametrize("split", [0, 512])
def test_attention_gate_pipelined(gpu, pipelined, split):
    RL.test_attention_gate(gpu, split)


@pytest.mark.parametrize("mode", ["bidir", "block_causal"])
def test_overflow_rerun_pipelined_d64(gpu, pipelined, mode):
    """The exact rerun (max-only pass, then the pipelined loop again with the
    true maximum) at head_dim 64."""
    spec = synth.AttnSpec(3, 32, 2, ("fixed", 0), 16, 4, 64)
    case = synth.make_attention_case(spec, 53, prefix_lens=[700, 3000, 96])
    case = A._plant_hot_keys(case, 54)
    for split in (0, 256):
        out = A.run_case(gpu, case, mode, kv_split_tokens=split)
        assert_attn_close(out, A.oracle_case(case, mode), f"rerun D=64 {mode} split={split}")
