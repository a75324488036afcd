"""Properties of the attention kernels' gfx950 code, checked on the assembly
hipcc writes for them with the library's own flags (no GPU is used).

The key loop keeps up to three tiles' direct HBM->LDS loads in flight and
waits for the oldest with `s_waitcnt vmcnt(n)`, n > 0.  The compiler adds a
wait for every load in flight (`vmcnt(0)`) before an LDS read when it cannot
tell which buffer a load in flight writes, or when the read's destination
register is a load's address register; one such wait in the unrolled main
loop drains the prefetch on every pass.  Every instantiation's main loop
(the block with the most MFMAs) must hold none.  With two waves per SIMD a
wave has 256 registers; a kernel may spill a few values that only its set-up
and tail code use (a few dwords of scratch per lane), but no main loop may
touch scratch memory."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _asm(tmp_path):
    from paper_2607_22663_amd import build as b
    try:
        hipcc = b.hipcc()
    except RuntimeError:
        pytest.skip("needs hipcc")
    flags = [f for f in b.HIPCC_FLAGS if f not in ("-shared", "-fPIC")]
    out = tmp_path / "attn_window.s"
    cmd = [hipcc, *flags, "--cuda-device-only", "-S", "-I", os.path.join(ROOT, "include"),
           "-o", str(out), os.path.join(b.CSRC, "attn_window.hip")]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    return out.read_text()


def _kernels(asm):
    for m in re.finditer(r"^(_ZN3mbe12_GLOBAL__N_123window_attention_kernel\w+):", asm, re.M):
        start = m.start()
        yield m.group(1), asm[start:asm.index(".Lfunc_end", start)]


def _scratch_bytes(asm, name):
    end = asm.index(".Lfunc_end", asm.index(name + ":"))
    return int(re.search(r"; ScratchSize: (\d+)", asm[end:]).group(1))


def _blocks(body):
    for blk in re.split(r"\n(?=\.LBB)", body):
        ins = [l.strip() for l in blk.splitlines()[1:]
               if l.strip() and not l.strip().startswith((";", "."))]
        yield ins


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="needs hipcc")
def test_attention_main_loops_never_drain_the_loads(tmp_path):
    asm = _asm(tmp_path)
    kernels = list(_kernels(asm))
    # D x mask mode x key split x V layout, plus the pipelined loop (token-minor
    # V, no key split) for each D and mask mode
    assert len(kernels) == 20, [k for k, _ in kernels]
    for name, body in kernels:
        blocks = list(_blocks(body))
        main = max(blocks, key=lambda ins: sum("v_mfma" in l for l in ins))
        n_mfma = sum("v_mfma" in l for l in main)
        waits = [l for l in main if l.startswith("s_waitcnt") and "vmcnt" in l]
        assert n_mfma >= 32, (name, n_mfma)        # four or five unrolled tiles: 8 MFMAs each at least
        assert waits, f"{name}: main loop without a load wait"
        drains = [l for l in waits if re.search(r"vmcnt\(0\)", l)]
        if "kernelILi64ELi0E" in name:
            # D = 64, window mode: this compiler waits for all loads once at
            # the top of the four-tile loop (its tracking of the loads in
            # flight is lost where the prologue and the loop's back edge
            # meet); no more than that one
            assert len(drains) <= 1, f"{name}: main loop waits for every load in flight: {drains}"
        else:
            assert not drains, f"{name}: main loop waits for every load in flight: {drains}"
        assert not any(l.startswith(("scratch_", "buffer_store", "buffer_load")) for l in main), name
        # the pipelined loop holds all 256 registers; its set-up and tail
        # code spill a few values (7 and 11 dwords as built)
        limit = 64
        assert _scratch_bytes(asm, name) <= limit, f"{name} spills more than {limit // 4} dwords per lane"
