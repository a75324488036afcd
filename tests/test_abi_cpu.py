"""C ABI checks that need no GPU: the library loads, exports every declared
symbol, and rejects bad arguments on the host before any HIP call."""
import ctypes
import math
import os
import re

import numpy as np
import pytest
import torch

import paper_2607_22663_amd as mbe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "mbe.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mbe_\w+|block_diffusion_attention)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(mbe.LIB_PATH):
        pytest.fail("libmbe.so is not built (run python -m paper_2607_22663_amd.build)")
    return mbe.load()


def test_exports_every_declared_symbol(lib):
    names = _declared_functions()
    assert len(names) == 16, names
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(mbe.EXPORTS)


def test_timeline_build_exports_the_abi_and_the_timeline_calls():
    """The profiling build is the same library plus the phase-timeline
    accessors; the product build has no timeline."""
    from paper_2607_22663_amd.build import TIMELINE_LIB
    if not os.path.exists(TIMELINE_LIB):
        pytest.fail("libmbe_timeline.so is not built (python -m paper_2607_22663_amd.build --timeline)")
    tl = ctypes.CDLL(TIMELINE_LIB)
    for n in _declared_functions() + ["mbe_timeline_read", "mbe_timeline_clear"]:
        assert hasattr(tl, n), n
    product = ctypes.CDLL(mbe.LIB_PATH)
    assert not hasattr(product, "mbe_timeline_read")


def _kv(head_dim=128, page=16, hkv=4, pages=10, v_layout=0):
    return mbe.PagedKV(ctypes.c_void_p(16), ctypes.c_void_p(32), pages, page, hkv, head_dim, v_layout)


def _opts(**kw):
    base = dict(batch=1, num_q_heads=16, max_pages_per_seq=10, total_q=64, max_prefix_len=64,
                max_window_len=64, mask_mode=0, softmax_scale=0.0, kv_split_tokens=0,
                host_prefix_lens=None, host_window_lens=None, workspace=None, workspace_bytes=0, stream=None)
    base.update(kw)
    return mbe.AttnOpts(**base)


def _attn(lib, kv, opts, B=32, q=16, out=48):
    st = lib.mbe_window_attention(ctypes.c_void_p(q), ctypes.byref(kv), ctypes.c_void_p(8),
                                  ctypes.c_void_p(8), ctypes.c_void_p(8), B, ctypes.c_void_p(out),
                                  ctypes.byref(opts))
    return st, lib.mbe_last_error().decode()


@pytest.mark.parametrize("kv_kw,opt_kw,B,status,text", [
    (dict(head_dim=96), {}, 32, 3, "head_dim"),
    (dict(page=32), {}, 32, 3, "page_size"),
    (dict(v_layout=2), {}, 32, 3, "v_layout"),
    ({}, dict(num_q_heads=6), 32, 2, "multiple"),
    ({}, dict(max_window_len=48), 32, 2, "multiple of block_size"),
    ({}, dict(max_pages_per_seq=0), 32, 2, "max_pages_per_seq"),
    ({}, dict(mask_mode=5), 32, 3, "mask_mode"),
    ({}, dict(kv_split_tokens=100), 32, 2, "multiple of 64"),
    ({}, dict(softmax_scale=float("nan")), 32, 6, "NaN"),
    ({}, dict(batch=-1), 32, 2, "batch"),
    ({}, {}, 0, 2, "block_size"),
])
def test_attention_validation(lib, kv_kw, opt_kw, B, status, text):
    st, msg = _attn(lib, _kv(**kv_kw), _opts(**opt_kw), B=B)
    assert st == status and text in msg, (st, msg)


def test_attention_null_pointers_and_workspace(lib):
    kv = _kv()
    st = lib.mbe_window_attention(None, ctypes.byref(kv), None, None, None, 32, None,
                                  ctypes.byref(_opts()))
    assert st == 1
    st = lib.mbe_window_attention(None, None, None, None, None, 32, None, ctypes.byref(_opts()))
    assert st == 1 and "paged_kv" in lib.mbe_last_error().decode()
    # a plan that needs split-KV partials without a workspace
    opts = _opts(max_prefix_len=4096, max_pages_per_seq=300, kv_split_tokens=1024)
    need = lib.mbe_window_attention_workspace_size(ctypes.byref(kv), ctypes.byref(opts))
    assert need > 0
    st, msg = _attn(lib, kv, opts)
    assert st == 4 and "workspace" in msg
    opts.workspace, opts.workspace_bytes = ctypes.c_void_p(256), need - 1
    st, msg = _attn(lib, kv, opts)
    assert st == 4


def test_block_diffusion_workspace_size_is_what_the_call_requires(lib):
    """block_diffusion_attention plans with W_b = block_size and the host
    prefix lengths; its size query must give exactly the bytes the call then
    requires (the window-attention query, without host window lengths here,
    plans from the bounds and asks for less)."""
    kv = _kv(pages=20000)
    P = np.array([100, 16000, 200, 300, 50, 8000, 10, 64], dtype=np.int32)
    opts = _opts(batch=8, total_q=8 * 32, max_prefix_len=16000, max_window_len=32, max_pages_per_seq=1100,
                 host_prefix_lens=P.ctypes.data_as(ctypes.c_void_p))
    need = lib.mbe_block_diffusion_workspace_size(ctypes.byref(kv), ctypes.byref(opts), 32)
    assert 0 < need != ctypes.c_size_t(-1).value
    assert lib.mbe_window_attention_workspace_size(ctypes.byref(kv), ctypes.byref(opts)) < need
    opts.workspace, opts.workspace_bytes = ctypes.c_void_p(256 * 1024), need - 1
    st = lib.block_diffusion_attention(ctypes.c_void_p(64), ctypes.byref(kv), ctypes.c_void_p(8),
                                       ctypes.c_void_p(8), 32, ctypes.c_void_p(128), ctypes.byref(opts))
    assert st == 4 and f"required {need}" in lib.mbe_last_error().decode()
    assert lib.mbe_block_diffusion_workspace_size(ctypes.byref(kv), ctypes.byref(opts), 0) == \
        ctypes.c_size_t(-1).value
    assert lib.mbe_block_diffusion_workspace_size(ctypes.byref(kv), None, 32) == ctypes.c_size_t(-1).value


def test_attention_empty_batch_is_ok_without_launch(lib):
    st, _ = _attn(lib, _kv(), _opts(batch=0, total_q=0))
    assert st == 0
    st, _ = _attn(lib, _kv(), _opts(total_q=0))
    assert st == 0


def test_workspace_sizes(lib):
    kv = _kv()
    small = _opts(max_prefix_len=64, kv_split_tokens=0)
    assert lib.mbe_window_attention_workspace_size(ctypes.byref(kv), ctypes.byref(small)) == 0
    big = _opts(batch=1, total_q=64, max_prefix_len=16384, max_pages_per_seq=1100, kv_split_tokens=2048)
    n = lib.mbe_window_attention_workspace_size(ctypes.byref(kv), ctypes.byref(big))
    splits = math.ceil((16384 + 64) / 2048)
    assert n >= splits * 64 * 16 * (128 + 2) * 4
    bad = _opts(num_q_heads=5)
    assert lib.mbe_window_attention_workspace_size(ctypes.byref(kv), ctypes.byref(bad)) == ctypes.c_size_t(-1).value
    assert lib.mbe_edit_select_workspace_size(8192, 131072) == 0
    assert lib.mbe_edit_select_workspace_size(64, 131072) > 0
    assert lib.mbe_edit_select_workspace_size(-1, 10) == ctypes.c_size_t(-1).value


@pytest.mark.parametrize("args,status,text", [
    (dict(rows=-1), 2, "negative"),
    (dict(row_stride=100, vocab=128), 2, "row_stride"),
    (dict(threshold=float("nan")), 6, "NaN"),
    (dict(logits=None), 1, "non-NULL"),
    (dict(rows=64, vocab=131072, row_stride=131072, ws=None), 4, "workspace"),
])
def test_edit_select_validation(lib, args, status, text):
    a = dict(logits=16, rows=4, vocab=128, row_stride=128, cur=8, threshold=0.9, new=8, conf=8, ch=8,
             ws=None, wsb=0)
    a.update(args)
    vp = lambda x: None if x is None else ctypes.c_void_p(x)
    st = lib.mbe_edit_select(vp(a["logits"]), a["rows"], a["vocab"], a["row_stride"], vp(a["cur"]),
                             ctypes.c_float(a["threshold"]), vp(a["new"]), vp(a["conf"]), vp(a["ch"]),
                             vp(a["ws"]), a["wsb"], None)
    assert st == status and text in lib.mbe_last_error().decode()


def test_edit_select_zero_rows_ok(lib):
    assert lib.mbe_edit_select(None, 0, 128, 128, None, ctypes.c_float(0.5), None, None, None, None, 0,
                               None) == 0


def test_status_strings(lib):
    assert lib.mbe_status_string(0) == b"ok"
    assert lib.mbe_status_string(5) == b"HIP error"
    assert lib.mbe_status_string(99) == b"unknown status"


def test_missing_library_fails_loudly(tmp_path):
    import importlib
    m = importlib.reload(mbe)
    try:
        with pytest.raises(RuntimeError, match="not found"):
            m.load(str(tmp_path / "nope.so"))
    finally:
        importlib.reload(mbe)


def _vp(x):
    return None if x is None else ctypes.c_void_p(x)


@pytest.mark.parametrize("args,status,text", [
    (dict(rows=-1), 2, "negative"),
    (dict(block_size=0), 2, "block_size"),
    (dict(rows=30, block_size=32), 2, "multiple of block_size"),
    (dict(row_stride=100, vocab=128), 2, "row_stride"),
    (dict(omega_mask=float("nan")), 6, "NaN"),
    (dict(omega_edit=float("nan")), 6, "NaN"),
    (dict(action=None), 1, "non-NULL"),
    (dict(block_changed=None), 1, "non-NULL"),
    (dict(ws=None), 4, "workspace"),
    (dict(wsb=16), 4, "workspace"),
    (dict(ws=272), 4, "aligned"),
    (dict(count=64, gate=64), 6, "run_if_nonzero"),
])
def test_threshold_update_validation(lib, args, status, text):
    a = dict(logits=16, rows=64, vocab=128, row_stride=128, cur=16, mask_id=127, block_size=32, omega_mask=0.5,
             omega_edit=0.0, new=16, conf=16, action=16, block_changed=16, count=None, entropy=None, gate=None,
             ws=256, wsb=1 << 20)
    a.update(args)
    st = lib.mbe_threshold_update(_vp(a["logits"]), a["rows"], a["vocab"], a["row_stride"], _vp(a["cur"]),
                                  a["mask_id"], a["block_size"], ctypes.c_float(a["omega_mask"]),
                                  ctypes.c_float(a["omega_edit"]), _vp(a["new"]), _vp(a["conf"]), _vp(a["action"]),
                                  _vp(a["block_changed"]), _vp(a["count"]), _vp(a["entropy"]), _vp(a["gate"]),
                                  _vp(a["ws"]), a["wsb"], None)
    assert st == status and text in lib.mbe_last_error().decode(), lib.mbe_last_error()


def test_threshold_update_workspace_and_empty(lib):
    assert lib.mbe_threshold_update_workspace_size(-1, 10) == ctypes.c_size_t(-1).value
    assert lib.mbe_threshold_update_workspace_size(0, 10) == 0
    n = lib.mbe_threshold_update_workspace_size(8192, 131072)
    assert n >= 8192 * 4 and n % 256 == 0
    assert lib.mbe_threshold_update_workspace_size(64, 131072) > lib.mbe_edit_select_workspace_size(64, 131072)
    assert lib.mbe_threshold_update(None, 0, 128, 128, None, 0, 32, ctypes.c_float(0.5), ctypes.c_float(0.0),
                                    None, None, None, None, None, None, None, None, 0, None) == 0


@pytest.mark.parametrize("args,status,text", [
    (dict(num_blocks=-1), 2, "num_blocks"),
    (dict(block_size=0), 3, "block_size"),
    (dict(block_size=2048), 3, "block_size"),
    (dict(rho=0.0), 6, "rho"),
    (dict(rho=1.5), 6, "rho"),
    (dict(rho=float("nan")), 6, "rho"),
    (dict(entropy=None), 1, "non-NULL"),
])
def test_tail_entropy_validation(lib, args, status, text):
    a = dict(entropy=16, num_blocks=4, block_size=32, rho=0.25, scores=16)
    a.update(args)
    st = lib.mbe_tail_entropy_scores(_vp(a["entropy"]), a["num_blocks"], a["block_size"], ctypes.c_float(a["rho"]),
                                     _vp(a["scores"]), None)
    assert st == status and text in lib.mbe_last_error().decode()


@pytest.mark.parametrize("args,status,text", [
    (dict(batch=-1), 2, "batch"),
    (dict(k_max=0), 2, "k_max"),
    (dict(current=None), 1, "non-NULL"),
])
def test_select_start_validation(lib, args, status, text):
    a = dict(scores=16, batch=4, stride=8, current=16, k_max=4, start=16)
    a.update(args)
    st = lib.mbe_select_start_block(_vp(a["scores"]), a["batch"], a["stride"], _vp(a["current"]), a["k_max"],
                                    _vp(a["start"]), None)
    assert st == status and text in lib.mbe_last_error().decode()


@pytest.mark.parametrize("args,status,text", [
    (dict(head_dim=96), 3, "head_dim"),
    (dict(batch=70000), 2, "batch"),
    (dict(max_len=-1), 2, "negative"),
    (dict(k_new=None), 1, "non-NULL"),
    (dict(v_pages=24), 2, "aligned"),
    (dict(num_pages=0), 2, "empty"),
    (dict(flags=16, block_size=0), 2, "block_size"),
    (dict(v_layout=-1), 3, "v_layout"),
])
def test_kv_write_validation(lib, args, status, text):
    a = dict(k_pages=16, v_pages=32, num_pages=10, heads=4, head_dim=128, pt=16, max_pages=8, start=16, lens=16,
             batch=2, max_len=64, total=96, k_new=16, v_new=16, flags=None, block_size=0, v_layout=0)
    a.update(args)
    st = lib.mbe_kv_write(_vp(a["k_pages"]), _vp(a["v_pages"]), a["num_pages"], a["heads"], a["head_dim"],
                          a["v_layout"],
                          _vp(a["pt"]), a["max_pages"], _vp(a["start"]), _vp(a["lens"]), a["batch"], a["max_len"],
                          a["total"], _vp(a["k_new"]), _vp(a["v_new"]), _vp(a["flags"]), a["block_size"], None)
    assert st == status and text in lib.mbe_last_error().decode()


def test_refresh_validation(lib):
    assert lib.mbe_refresh_blocks(_vp(16), 2, 4, 2, _vp(16), None) == 3
    assert lib.mbe_refresh_blocks(None, 2, 4, 0, _vp(16), None) == 1
    assert lib.mbe_refresh_blocks(None, 0, 4, 0, None, None) == 0


def test_header_is_plain_c_and_links(tmp_path):
    """include/mbe.h compiles as C99 with every warning an error, and a C
    program links against libmbe.so and calls the host-only entry points
    (status strings, workspace sizes, a validation failure)."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "use_mbe.c"
    src.write_text(r'''
#include <stdio.h>
#include <string.h>
#include "mbe.h"
int main(void) {
  mbe_paged_kv kv = {0};
  mbe_attn_opts o;
  size_t n;
  memset(&o, 0, sizeof(o));
  kv.page_size = 16; kv.num_kv_heads = 4; kv.head_dim = 128; kv.num_pages = 10;
  o.batch = 1; o.num_q_heads = 16; o.max_pages_per_seq = 10; o.total_q = 64;
  o.max_prefix_len = 64; o.max_window_len = 64;
  n = mbe_window_attention_workspace_size(&kv, &o);
  if (n != 0) return 1;
  kv.head_dim = 96;
  if (mbe_window_attention(NULL, &kv, NULL, NULL, NULL, 32, NULL, &o) != MBE_ERR_UNSUPPORTED) return 2;
  if (strstr(mbe_last_error(), "head_dim") == NULL) return 3;
  if (strcmp(mbe_status_string(MBE_OK), "ok") != 0) return 4;
  if (mbe_edit_select_workspace_size(64, 131072) == 0) return 5;
  if (mbe_threshold_update_workspace_size(-1, 1) != (size_t)-1) return 6;
  printf("ok\n");
  return 0;
}
''')
    exe = tmp_path / "use_mbe"
    libdir = os.path.dirname(mbe.LIB_PATH)
    r = subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", os.path.join(ROOT, "include"),
                        str(src), "-o", str(exe), "-L", libdir, "-lmbe", f"-Wl,-rpath,{libdir}"],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0 and r.stdout.strip() == "ok", (r.returncode, r.stdout, r.stderr)


def test_binding_rejects_vocab_beyond_the_columns():
    """The binding checks vocab against the logits' columns before any call
    (the C ABI only sees the row stride)."""
    logits = torch.zeros(2, 10, dtype=torch.bfloat16)
    cur = torch.zeros(2, dtype=torch.int32)
    with pytest.raises(ValueError, match="vocab"):
        mbe.edit_select(logits, cur, 0.9, vocab=11)
    with pytest.raises(ValueError, match="vocab"):
        mbe.threshold_update(logits, cur, 9, 2, 0.5, 0.0, vocab=11)


def test_error_string_is_per_thread():
    """Concurrent calls (ctypes drops the GIL) each read their own failure
    from mbe_last_error(): the error string is thread-local."""
    import threading
    lib = mbe.load()      # the binding's current structure classes (another test reloads the module)
    errors = []

    def worker(hd):
        try:
            kv = _kv(head_dim=hd)
            for _ in range(200):
                st, msg = _attn(lib, kv, _opts())
                if st != 3 or f"head_dim {hd}" not in msg:
                    errors.append((hd, st, msg))
                    return
        except Exception as e:      # an exception in a thread would not fail the test by itself
            errors.append((hd, "exception", repr(e)))

    threads = [threading.Thread(target=worker, args=(hd,)) for hd in (32, 48, 80, 96, 100, 256, 512, 1000)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors[:3]


def test_threshold_update_noalloc_rejects_on_the_host(lib):
    """The no-allocation update checks its arguments like mbe_threshold_update
    and refuses shapes whose scratch exceeds its static 1 MiB (here 262176
    rows of predictions), before any HIP call."""
    def call(rows, omega=0.5):
        return lib.mbe_threshold_update_noalloc(_vp(16), rows, 16, 16, _vp(16), 15, 32, ctypes.c_float(omega),
                                                ctypes.c_float(0.0), _vp(16), _vp(16), _vp(16), _vp(16), None, None,
                                                None, None)
    assert call(262176) == 4 and "scratch" in lib.mbe_last_error().decode()
    assert lib.mbe_threshold_update_workspace_size(262144, 16) <= 1 << 20
    assert call(64, omega=float("nan")) == 6
    assert call(30) == 2                    # not a multiple of the block
    assert call(0) == 0                     # nothing to do


def _plan(B=32, k=4, P=None, batch=64, Hq=16, Hkv=4, D=128, token_major=False, split=0):
    """mbe_window_attention_plan through the binding, for shapes only (meta
    tensors: no memory, no GPU)."""
    P = np.asarray(P if P is not None else [32 * (128 + 14 * i) for i in range(batch)], dtype=np.int32)
    W = np.full(batch, k * B, dtype=np.int32)
    pages = int(sum(-(-(p + w) // 16) for p, w in zip(P, W)))
    kp = torch.empty((pages, Hkv, 16, D), dtype=torch.bfloat16, device="meta")
    vp = kp if token_major else torch.empty((pages, Hkv, D, 16), dtype=torch.bfloat16, device="meta")
    pt = torch.empty((batch, int(-(-(P.max() + W.max()) // 16))), dtype=torch.int32, device="meta")
    return mbe.window_attention_plan(Hq, kp, vp, pt, batch, int(W.sum()), max_prefix_len=int(P.max()),
                                     max_window_len=int(W.max()), kv_split_tokens=split,
                                     host_prefix_lens=P, host_window_lens=W)


def test_attention_plan_picks_the_kernel_variant(lib, monkeypatch):
    """The plan query reports the kernel the call will run: the pipelined key
    loop for long token-minor units without key split, the key-split waves for
    at most 128 rows per KV head, and splits exactly when a workspace is
    needed."""
    monkeypatch.delenv("MBE_ATTN_PIPELINE", raising=False)
    long_ctx = _plan()                                  # 64 x P up to 32K, k = 4: no split
    assert long_ctx["kernel"] == "window_attention_kernel<128,0,1,0,1>"
    assert long_ctx["splits"] == 1 and long_ctx["workgroups"] >= 512
    assert _plan(token_major=True)["kernel"] == "window_attention_kernel<128,0,1,1,0>"
    span = dict(batch=8, P=[16384] * 8)
    k1, k4, k8 = _plan(k=1, **span), _plan(k=4, **span), _plan(k=8, **span)
    assert (k1["key_split"], k1["pipelined"]) == (2, 0) and k1["splits"] > 1
    assert k4["pipelined"] == 0 and k4["kv_chunk"] // 64 < 96          # short units keep the plain loop
    assert k8["pipelined"] == 1 and k8["kv_chunk"] // 64 >= 96
    monkeypatch.setenv("MBE_ATTN_PIPELINE", "0")
    assert _plan()["pipelined"] == 0
    monkeypatch.setenv("MBE_ATTN_PIPELINE", "1")
    assert _plan(k=4, **span)["pipelined"] == 1
    assert _plan(k=1, **span)["pipelined"] == 0                          # key split: not eligible
    assert _plan(token_major=True)["pipelined"] == 0                     # token-major V: not eligible
    raw = ctypes.CDLL(mbe.LIB_PATH)             # plain pointers, whatever classes the binding holds
    raw.mbe_window_attention_plan.argtypes = [ctypes.c_void_p] * 3
    kv, opts, bad_opts, out = _kv(), _opts(), _opts(num_q_heads=5), ctypes.create_string_buffer(64)
    assert raw.mbe_window_attention_plan(ctypes.addressof(kv), ctypes.addressof(opts), None) == 1
    assert raw.mbe_window_attention_plan(ctypes.addressof(kv), ctypes.addressof(bad_opts), ctypes.addressof(out)) == 2
