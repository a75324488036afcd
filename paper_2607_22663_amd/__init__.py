"""Python binding of libmbe, the MBE editing-pass hot path on MI355X (gfx950).

Argument marshalling only: every step of the path runs in the HIP kernels of
libmbe.so, called through its C ABI (include/mbe.h) with ctypes.  PyTorch
provides device memory and the current stream.  If libmbe.so is missing or
cannot be loaded, every call raises; there is no other implementation.

    window_attention(q, k_pages, v_pages, page_table, prefix_lens, window_lens, block_size)
    block_diffusion_attention(q, k_pages, v_pages, page_table, prefix_lens, block_size)
    edit_select(logits, cur_tokens, threshold) -> (new_tokens, conf, changed_mask)
"""
from __future__ import annotations

import ctypes
import functools
import os
import threading
from typing import Optional

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmbe.so")

MBE_OK = 0
STATUS_NAMES = {0: "MBE_OK", 1: "MBE_ERR_NULL_ARG", 2: "MBE_ERR_BAD_SHAPE", 3: "MBE_ERR_UNSUPPORTED",
                4: "MBE_ERR_WORKSPACE", 5: "MBE_ERR_HIP", 6: "MBE_ERR_BAD_VALUE"}
MASK_MODES = {"bidir": 0, "block_causal": 1}

EXPORTS = ("mbe_window_attention", "block_diffusion_attention", "mbe_window_attention_workspace_size",
           "mbe_block_diffusion_workspace_size", "mbe_edit_select", "mbe_edit_select_workspace_size",
           "mbe_threshold_update", "mbe_threshold_update_workspace_size", "mbe_tail_entropy_scores",
           "mbe_select_start_block", "mbe_kv_write", "mbe_refresh_blocks", "mbe_status_string", "mbe_last_error",
           "mbe_threshold_update_noalloc", "mbe_window_attention_plan")
ACTIONS = {"keep": 0, "unmask": 1, "force_unmask": 2, "edit": 3}
REFRESH_MODES = {"changed": 0, "changed_and_later": 1}


class MbeError(RuntimeError):
    def __init__(self, call, status, detail):
        self.status = status
        super().__init__(f"{call}: {STATUS_NAMES.get(status, status)}: {detail}")


V_TOKEN_MINOR, V_TOKEN_MAJOR = 0, 1


class PagedKV(ctypes.Structure):
    _fields_ = [("k_pages", ctypes.c_void_p), ("v_pages", ctypes.c_void_p),
                ("num_pages", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("v_layout", ctypes.c_int32)]


def v_layout_of(k_pages, v_pages):
    """V_TOKEN_MAJOR when v_pages is [num_pages, Hkv, 16, D] like k_pages,
    V_TOKEN_MINOR when it is [num_pages, Hkv, D, 16] (head_dim is never 16)."""
    n_pages, hkv, page, d = k_pages.shape
    if tuple(v_pages.shape) == (n_pages, hkv, page, d):
        return V_TOKEN_MAJOR
    if tuple(v_pages.shape) == (n_pages, hkv, d, page):
        return V_TOKEN_MINOR
    raise ValueError(f"v_pages must be [num_pages, Hkv, 16, D] or [num_pages, Hkv, D, 16] = "
                     f"{(n_pages, hkv, page, d)} or {(n_pages, hkv, d, page)}, got {tuple(v_pages.shape)}")


class AttnOpts(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("max_pages_per_seq", ctypes.c_int32), ("total_q", ctypes.c_int32),
                ("max_prefix_len", ctypes.c_int32), ("max_window_len", ctypes.c_int32),
                ("mask_mode", ctypes.c_int32), ("softmax_scale", ctypes.c_float),
                ("kv_split_tokens", ctypes.c_int32), ("host_prefix_lens", ctypes.c_void_p),
                ("host_window_lens", ctypes.c_void_p), ("workspace", ctypes.c_void_p),
                ("workspace_bytes", ctypes.c_size_t), ("stream", ctypes.c_void_p),
                ("block_flags", ctypes.c_void_p), ("run_if_nonzero", ctypes.c_void_p)]


class AttnPlan(ctypes.Structure):
    _fields_ = [("splits", ctypes.c_int32), ("kv_chunk", ctypes.c_int32), ("key_split", ctypes.c_int32),
                ("pipelined", ctypes.c_int32), ("workgroups", ctypes.c_int64)]


_lib = None
_lock = threading.Lock()


def load(path: Optional[str] = None) -> ctypes.CDLL:
    """Loads libmbe.so (once).  Raises if it is missing or lacks a symbol."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        p = path or LIB_PATH
        if not os.path.exists(p):
            raise RuntimeError(f"{p} not found: build it with `python -m paper_2607_22663_amd.build`")
        lib = ctypes.CDLL(p)
        for name in EXPORTS:
            if not hasattr(lib, name):
                raise RuntimeError(f"{p} does not export {name}")
        vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        lib.mbe_window_attention.argtypes = [vp, ctypes.POINTER(PagedKV), vp, vp, vp, i32, vp,
                                             ctypes.POINTER(AttnOpts)]
        lib.mbe_window_attention.restype = ctypes.c_int
        lib.block_diffusion_attention.argtypes = [vp, ctypes.POINTER(PagedKV), vp, vp, i32, vp,
                                                  ctypes.POINTER(AttnOpts)]
        lib.block_diffusion_attention.restype = ctypes.c_int
        lib.mbe_window_attention_workspace_size.argtypes = [ctypes.POINTER(PagedKV), ctypes.POINTER(AttnOpts)]
        lib.mbe_window_attention_workspace_size.restype = sz
        lib.mbe_window_attention_plan.argtypes = [ctypes.POINTER(PagedKV), ctypes.POINTER(AttnOpts),
                                                  ctypes.POINTER(AttnPlan)]
        lib.mbe_window_attention_plan.restype = ctypes.c_int
        lib.mbe_block_diffusion_workspace_size.argtypes = [ctypes.POINTER(PagedKV), ctypes.POINTER(AttnOpts), i32]
        lib.mbe_block_diffusion_workspace_size.restype = sz
        lib.mbe_edit_select.argtypes = [vp, i64, i64, i64, vp, ctypes.c_float, vp, vp, vp, vp, sz, vp]
        lib.mbe_edit_select.restype = ctypes.c_int
        lib.mbe_edit_select_workspace_size.argtypes = [i64, i64]
        lib.mbe_edit_select_workspace_size.restype = sz
        f32 = ctypes.c_float
        lib.mbe_threshold_update.argtypes = [vp, i64, i64, i64, vp, i32, i32, f32, f32, vp, vp, vp, vp, vp, vp, vp,
                                             vp, sz, vp]
        lib.mbe_threshold_update.restype = ctypes.c_int
        lib.mbe_threshold_update_noalloc.argtypes = [vp, i64, i64, i64, vp, i32, i32, f32, f32, vp, vp, vp, vp, vp,
                                                     vp, vp, vp]
        lib.mbe_threshold_update_noalloc.restype = ctypes.c_int
        lib.mbe_threshold_update_workspace_size.argtypes = [i64, i64]
        lib.mbe_threshold_update_workspace_size.restype = sz
        lib.mbe_tail_entropy_scores.argtypes = [vp, i64, i32, f32, vp, vp]
        lib.mbe_tail_entropy_scores.restype = ctypes.c_int
        lib.mbe_select_start_block.argtypes = [vp, i32, i32, vp, i32, vp, vp]
        lib.mbe_select_start_block.restype = ctypes.c_int
        lib.mbe_kv_write.argtypes = [vp, vp, i32, i32, i32, i32, vp, i32, vp, vp, i32, i32, i32, vp, vp, vp, i32, vp]
        lib.mbe_kv_write.restype = ctypes.c_int
        lib.mbe_refresh_blocks.argtypes = [vp, i32, i32, i32, vp, vp]
        lib.mbe_refresh_blocks.restype = ctypes.c_int
        lib.mbe_status_string.argtypes = [ctypes.c_int]
        lib.mbe_status_string.restype = ctypes.c_char_p
        lib.mbe_last_error.argtypes = []
        lib.mbe_last_error.restype = ctypes.c_char_p
        _lib = lib
        return lib


def _on_device(fn):
    """Runs a call with the current HIP device set to the device of its first
    (tensor) argument: the library launches on the current device."""
    @functools.wraps(fn)
    def wrapper(*args, **kwargs):
        t = args[0] if args else None
        if isinstance(t, torch.Tensor) and t.is_cuda and t.device.index != torch.cuda.current_device():
            with torch.cuda.device(t.device):
                return fn(*args, **kwargs)
        return fn(*args, **kwargs)
    return wrapper


def _check(call, status):
    if status != MBE_OK:
        raise MbeError(call, status, load().mbe_last_error().decode(errors="replace"))


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _need(t: torch.Tensor, name: str, dtype, device, ndim=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.device != device:
        raise ValueError(f"{name} must be on {device}, got {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions, got {t.dim()}")


_workspaces = {}


def _workspace(kind: str, device: torch.device, nbytes: int) -> Optional[torch.Tensor]:
    """Per-(kind, device, current stream) workspace, grown on demand (contents
    do not matter).  Calls on one stream run in order, so they may share it;
    calls on different streams get different buffers and never race."""
    if nbytes == 0:
        return None
    key = (kind, device.index, torch.cuda.current_stream(device).cuda_stream)
    ws = _workspaces.get(key)
    if ws is None or ws.numel() < nbytes:
        ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
        _workspaces[key] = ws
    return ws


MBE_ERR_WORKSPACE = 4


def _call_with_workspace(call, size, opts, device, workspace):
    """Runs an attention call whose split plan may need a workspace.  With a
    caller's workspace, that one.  Otherwise the shared workspace of this
    stream as it is, first: only when the library reports it too small (or
    absent) is the size queried, the workspace grown and the call repeated, so
    a steady stream of calls plans once per call."""
    if workspace is not None:
        if workspace.dtype != torch.uint8 or not workspace.is_cuda:
            raise ValueError("workspace must be a uint8 device tensor")
        opts.workspace, opts.workspace_bytes = _ptr(workspace), workspace.numel()
        return call()
    key = ("attn", device.index, torch.cuda.current_stream(device).cuda_stream)
    ws = _workspaces.get(key)
    opts.workspace, opts.workspace_bytes = (_ptr(ws), ws.numel()) if ws is not None else (None, 0)
    status = call()
    if status != MBE_ERR_WORKSPACE:
        return status
    need = size()
    if need == ctypes.c_size_t(-1).value:
        return status
    ws = _workspace("attn", device, need)
    opts.workspace, opts.workspace_bytes = (_ptr(ws), need) if ws is not None else (None, 0)
    return call()


def _own_workspace(ws: torch.Tensor, need: int) -> Optional[torch.Tensor]:
    if need == 0:
        return None
    if ws.dtype != torch.uint8 or not ws.is_cuda or ws.numel() < need:
        raise ValueError(f"workspace must be a uint8 device tensor of at least {need} bytes")
    return ws


def workspace_bytes_threshold_update(rows, vocab):
    n = load().mbe_threshold_update_workspace_size(int(rows), int(vocab))
    return 0 if n == ctypes.c_size_t(-1).value else n


def workspace_bytes_window_attention(q, k_pages, page_table, batch, *, max_prefix_len,
                                     max_window_len, mask_mode="bidir", kv_split_tokens=0):
    """Workspace bytes of a window_attention call planned from bounds only
    (no host lengths), as a captured graph replays it."""
    lib = load()
    kv = PagedKV(None, None, k_pages.shape[0], k_pages.shape[2], k_pages.shape[1], k_pages.shape[3], 0)
    opts = AttnOpts(int(batch), q.shape[1], page_table.shape[1], q.shape[0], int(max_prefix_len), int(max_window_len),
                    MASK_MODES[mask_mode] if isinstance(mask_mode, str) else int(mask_mode), 0.0,
                    int(kv_split_tokens), None, None, None, 0, None, None, None)
    n = lib.mbe_window_attention_workspace_size(ctypes.byref(kv), ctypes.byref(opts))
    if n == ctypes.c_size_t(-1).value:
        raise ValueError("invalid attention shapes")
    return n


def window_attention_plan(num_q_heads, k_pages, v_pages, page_table, batch, total_q, *, max_prefix_len,
                          max_window_len, mask_mode="bidir", kv_split_tokens=0, host_prefix_lens=None,
                          host_window_lens=None):
    """The launch plan a window_attention call with these shapes makes (host
    only): dict of splits, kv_chunk, key_split, pipelined, workgroups, and the
    main kernel's name as rocprofv3 reports it (window_attention_kernel<D,
    MODE, KS, VT, PIPE>)."""
    lib = load()
    layout = v_layout_of(k_pages, v_pages)
    kv = PagedKV(None, None, k_pages.shape[0], k_pages.shape[2], k_pages.shape[1], k_pages.shape[3], layout)
    hp = _host_i32(host_prefix_lens, batch, "host_prefix_lens")
    hw = _host_i32(host_window_lens, batch, "host_window_lens")
    mode = MASK_MODES[mask_mode] if isinstance(mask_mode, str) else int(mask_mode)
    opts = AttnOpts(int(batch), int(num_q_heads), page_table.shape[1], int(total_q), int(max_prefix_len),
                    int(max_window_len), mode, 0.0, int(kv_split_tokens), _ptr(hp), _ptr(hw), None, 0, None,
                    None, None)
    plan = AttnPlan()
    _check("mbe_window_attention_plan", lib.mbe_window_attention_plan(ctypes.byref(kv), ctypes.byref(opts),
                                                                      ctypes.byref(plan)))
    d = {f: getattr(plan, f) for f, _ in AttnPlan._fields_}
    d["kernel"] = (f"window_attention_kernel<{k_pages.shape[3]},{mode},{plan.key_split},"
                   f"{int(layout == V_TOKEN_MAJOR)},{plan.pipelined}>")
    return d


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _attn_common(q, k_pages, v_pages, page_table, prefix_lens, out):
    dev = q.device
    _need(q, "q", torch.bfloat16, dev, 3)
    _need(k_pages, "k_pages", torch.bfloat16, dev, 4)
    _need(v_pages, "v_pages", torch.bfloat16, dev, 4)
    _need(page_table, "page_table", torch.int32, dev, 2)
    _need(prefix_lens, "prefix_lens", torch.int32, dev, 1)
    n_pages, hkv, page, d = k_pages.shape
    layout = v_layout_of(k_pages, v_pages)
    if q.shape[2] != d:
        raise ValueError(f"q head_dim {q.shape[2]} != cache head_dim {d}")
    if page_table.shape[0] != prefix_lens.shape[0]:
        raise ValueError("page_table and prefix_lens disagree on the batch size")
    if out is None:
        out = torch.empty_like(q)
    else:
        _need(out, "out", torch.bfloat16, dev, 3)
        if out.shape != q.shape:
            raise ValueError("out must have the shape of q")
    kv = PagedKV(_ptr(k_pages), _ptr(v_pages), n_pages, page, hkv, d, layout)
    return kv, out


def _flags_gate(block_flags, shape, gate, device):
    if block_flags is not None:
        _need(block_flags, "block_flags", torch.uint8, device, 2)
        if tuple(block_flags.shape) != tuple(shape):
            raise ValueError(f"block_flags must be {tuple(shape)}, got {tuple(block_flags.shape)}")
    if gate is not None:
        _need(gate, "run_if_nonzero", torch.int32, device)
        if gate.numel() < 1:
            raise ValueError("run_if_nonzero must hold one int32")


def _host_i32(x, batch, name):
    """A contiguous host int32 copy (kept alive by the caller) or None."""
    if x is None:
        return None
    a = torch.as_tensor(x, dtype=torch.int32, device="cpu").contiguous()
    if a.numel() != batch:
        raise ValueError(f"{name} must have {batch} entries")
    return a


@_on_device
def window_attention(q, k_pages, v_pages, page_table, prefix_lens, window_lens, block_size, *,
                     out=None, mask_mode="bidir", softmax_scale=None, max_prefix_len=None,
                     max_window_len=None, kv_split_tokens=0, host_prefix_lens=None, host_window_lens=None,
                     workspace=None, block_flags=None, run_if_nonzero=None):
    """MBE editing-window attention (paper, Sec. "Training-Free MBE Decoding",
    Eq. (4)).  Layouts as in include/mbe.h; the V pool's layout is read from
    its shape (v_layout_of).

    max_prefix_len / max_window_len are host-side bounds.  host_prefix_lens /
    host_window_lens are optional host copies of the lengths (they let the
    library size splits from the total work and start long sequences first).
    When neither bounds nor host lengths are given, the lengths are copied
    from the device (a synchronisation).  workspace: an optional caller-owned
    uint8 device tensor used instead of the module's shared one (as a
    captured graph needs).  block_flags: optional uint8 [batch,
    max_window_len / block_size] device tensor; only the rows of flagged
    window blocks are computed and written (targeted refresh).
    run_if_nonzero: optional int32 [1] device tensor; the call does nothing
    when it holds 0 (e.g. the previous editing pass's changed count)."""
    lib = load()
    kv, out = _attn_common(q, k_pages, v_pages, page_table, prefix_lens, out)
    _need(window_lens, "window_lens", torch.int32, q.device, 1)
    batch = prefix_lens.shape[0]
    if max_prefix_len is None and host_prefix_lens is None:
        host_prefix_lens = prefix_lens.cpu()
    if max_window_len is None and host_window_lens is None:
        host_window_lens = window_lens.cpu()
    hp = _host_i32(host_prefix_lens, batch, "host_prefix_lens")
    hw = _host_i32(host_window_lens, batch, "host_window_lens")
    if max_prefix_len is None:
        max_prefix_len = int(hp.max()) if batch else 0
    if max_window_len is None:
        max_window_len = int(hw.max()) if batch else 0
    stream = _stream(q.device)
    nblk = int(max_window_len) // int(block_size) if int(block_size) > 0 else 0
    _flags_gate(block_flags, (batch, nblk), run_if_nonzero, q.device)
    opts = AttnOpts(batch, q.shape[1], page_table.shape[1], q.shape[0], int(max_prefix_len),
                    int(max_window_len), MASK_MODES[mask_mode] if isinstance(mask_mode, str) else int(mask_mode),
                    float(softmax_scale or 0.0), int(kv_split_tokens), _ptr(hp), _ptr(hw), None, 0, stream,
                    _ptr(block_flags), _ptr(run_if_nonzero))
    def call():
        return lib.mbe_window_attention(_ptr(q), ctypes.byref(kv), _ptr(page_table), _ptr(prefix_lens),
                                        _ptr(window_lens), int(block_size), _ptr(out), ctypes.byref(opts))

    def size():
        return lib.mbe_window_attention_workspace_size(ctypes.byref(kv), ctypes.byref(opts))

    _check("mbe_window_attention", _call_with_workspace(call, size, opts, q.device, workspace))
    return out


@_on_device
def block_diffusion_attention(q, k_pages, v_pages, page_table, prefix_lens, block_size, *,
                              out=None, softmax_scale=None, max_prefix_len=None, kv_split_tokens=0,
                              host_prefix_lens=None, block_flags=None, run_if_nonzero=None):
    """Standard single-block step (paper, Sec. "Block diffusion"): q holds
    block_size rows per sequence."""
    lib = load()
    kv, out = _attn_common(q, k_pages, v_pages, page_table, prefix_lens, out)
    batch = prefix_lens.shape[0]
    if max_prefix_len is None and host_prefix_lens is None:
        host_prefix_lens = prefix_lens.cpu()
    hp = _host_i32(host_prefix_lens, batch, "host_prefix_lens")
    if max_prefix_len is None:
        max_prefix_len = int(hp.max()) if batch else 0
    stream = _stream(q.device)
    _flags_gate(block_flags, (batch, 1), run_if_nonzero, q.device)
    opts = AttnOpts(batch, q.shape[1], page_table.shape[1], q.shape[0], int(max_prefix_len),
                    int(block_size), 0, float(softmax_scale or 0.0), int(kv_split_tokens), _ptr(hp), None,
                    None, 0, stream, _ptr(block_flags), _ptr(run_if_nonzero))
    def call():
        return lib.block_diffusion_attention(_ptr(q), ctypes.byref(kv), _ptr(page_table), _ptr(prefix_lens),
                                             int(block_size), _ptr(out), ctypes.byref(opts))

    def size():
        return lib.mbe_block_diffusion_workspace_size(ctypes.byref(kv), ctypes.byref(opts), int(block_size))

    _check("block_diffusion_attention", _call_with_workspace(call, size, opts, q.device, None))
    return out


@_on_device
def edit_select(logits, cur_tokens, threshold, *, vocab=None, out=None):
    """Edit selection (paper, Eq. (1), token-to-token set).  logits: bf16
    [rows, row_stride] (the first `vocab` columns are used; default all).
    Returns (new_tokens int32, conf float32, changed_mask uint8)."""
    lib = load()
    dev = logits.device
    _need(cur_tokens, "cur_tokens", torch.int32, dev, 1)
    if logits.dtype != torch.bfloat16 or logits.dim() != 2 or logits.stride(1) != 1:
        raise ValueError("logits must be a bf16 [rows, row_stride] tensor with unit column stride")
    rows = logits.shape[0]
    if cur_tokens.shape[0] != rows:
        raise ValueError("cur_tokens must have one entry per row")
    v = logits.shape[1] if vocab is None else int(vocab)
    if not 0 <= v <= logits.shape[1]:
        raise ValueError(f"vocab {v} outside [0, {logits.shape[1]}] (the columns of logits)")
    ld = logits.stride(0) if rows > 1 else max(logits.shape[1], 1)
    if out is None:
        new = torch.empty(rows, dtype=torch.int32, device=dev)
        conf = torch.empty(rows, dtype=torch.float32, device=dev)
        changed = torch.empty(rows, dtype=torch.uint8, device=dev)
    else:
        new, conf, changed = out
    stream = _stream(dev)
    need = lib.mbe_edit_select_workspace_size(rows, v)
    ws = _workspace("edit", dev, need if need != ctypes.c_size_t(-1).value else 0)
    _check("mbe_edit_select", lib.mbe_edit_select(
        _ptr(logits), rows, v, ld, _ptr(cur_tokens), ctypes.c_float(threshold), _ptr(new), _ptr(conf),
        _ptr(changed), _ptr(ws), need if ws is not None else 0, stream))
    return new, conf, changed


@_on_device
def threshold_update(logits, cur_tokens, mask_id, block_size, omega_mask, omega_edit, *, vocab=None,
                     with_entropy=False, out=None, workspace=None, run_if_nonzero=None):
    """Full threshold update (paper, Eq. (1) with force-unmask).  Rows form
    blocks of block_size consecutive rows.  Returns a dict of device tensors:
    new_tokens int32, conf float32, action uint8 (ACTIONS), block_changed
    uint8 [rows / block_size], changed_count int32 [1] and, when asked,
    entropy float32 (nats).  out["new_tokens"] may be cur_tokens itself (in
    place).  run_if_nonzero: optional int32 device tensor (not
    out["changed_count"]); when it holds 0 the pass keeps every row."""
    lib = load()
    dev = logits.device
    _need(cur_tokens, "cur_tokens", torch.int32, dev, 1)
    if logits.dtype != torch.bfloat16 or logits.dim() != 2 or logits.stride(1) != 1:
        raise ValueError("logits must be a bf16 [rows, row_stride] tensor with unit column stride")
    rows = logits.shape[0]
    if cur_tokens.shape[0] != rows:
        raise ValueError("cur_tokens must have one entry per row")
    v = logits.shape[1] if vocab is None else int(vocab)
    if not 0 <= v <= logits.shape[1]:
        raise ValueError(f"vocab {v} outside [0, {logits.shape[1]}] (the columns of logits)")
    ld = logits.stride(0) if rows > 1 else max(logits.shape[1], 1)
    nblk = rows // block_size if block_size > 0 else 0
    if out is None:
        out = {"new_tokens": torch.empty(rows, dtype=torch.int32, device=dev),
               "conf": torch.empty(rows, dtype=torch.float32, device=dev),
               "action": torch.empty(rows, dtype=torch.uint8, device=dev),
               "block_changed": torch.empty(max(nblk, 1), dtype=torch.uint8, device=dev),
               "changed_count": torch.empty(1, dtype=torch.int32, device=dev)}
        if with_entropy:
            out["entropy"] = torch.empty(rows, dtype=torch.float32, device=dev)
    need = lib.mbe_threshold_update_workspace_size(rows, v)
    need = need if need != ctypes.c_size_t(-1).value else 0
    ws = _workspace("update", dev, need) if workspace is None else _own_workspace(workspace, need)
    _flags_gate(None, None, run_if_nonzero, dev)
    _check("mbe_threshold_update", lib.mbe_threshold_update(
        _ptr(logits), rows, v, ld, _ptr(cur_tokens), int(mask_id), int(block_size), ctypes.c_float(omega_mask),
        ctypes.c_float(omega_edit), _ptr(out["new_tokens"]), _ptr(out["conf"]), _ptr(out["action"]),
        _ptr(out["block_changed"]), _ptr(out.get("changed_count")), _ptr(out.get("entropy")), _ptr(run_if_nonzero),
        _ptr(ws), need if ws is not None else 0, _stream(dev)))
    return out


@_on_device
def threshold_update_noalloc(logits, cur_tokens, mask_id, block_size, omega_mask, omega_edit, *, out,
                             vocab=None, run_if_nonzero=None):
    """threshold_update through mbe_threshold_update_noalloc: no workspace and
    no allocation (the library's static per-GPU scratch).  `out` is the dict
    of output tensors threshold_update returns (entropy and changed_count
    optional); nothing is allocated here either."""
    lib = load()
    dev = logits.device
    _need(cur_tokens, "cur_tokens", torch.int32, dev, 1)
    if logits.dtype != torch.bfloat16 or logits.dim() != 2 or logits.stride(1) != 1:
        raise ValueError("logits must be a bf16 [rows, row_stride] tensor with unit column stride")
    rows = logits.shape[0]
    v = logits.shape[1] if vocab is None else int(vocab)
    if cur_tokens.shape[0] != rows or not 0 <= v <= logits.shape[1]:
        raise ValueError("cur_tokens must have one entry per row and vocab fit the columns")
    ld = logits.stride(0) if rows > 1 else max(logits.shape[1], 1)
    _flags_gate(None, None, run_if_nonzero, dev)
    _check("mbe_threshold_update_noalloc", lib.mbe_threshold_update_noalloc(
        _ptr(logits), rows, v, ld, _ptr(cur_tokens), int(mask_id), int(block_size), ctypes.c_float(omega_mask),
        ctypes.c_float(omega_edit), _ptr(out["new_tokens"]), _ptr(out["conf"]), _ptr(out["action"]),
        _ptr(out["block_changed"]), _ptr(out.get("changed_count")), _ptr(out.get("entropy")), _ptr(run_if_nonzero),
        _stream(dev)))
    return out


@_on_device
def tail_entropy_scores(entropy, block_size, rho, *, out=None):
    """Eq. (5): mean of the ceil(rho * B) largest entropies of every block of
    block_size consecutive rows.  entropy: float32 [num_blocks * B]."""
    lib = load()
    dev = entropy.device
    _need(entropy, "entropy", torch.float32, dev, 1)
    nblk = entropy.shape[0] // block_size if block_size > 0 else 0
    scores = torch.empty(nblk, dtype=torch.float32, device=dev) if out is None else out
    _check("mbe_tail_entropy_scores", lib.mbe_tail_entropy_scores(
        _ptr(entropy), nblk, int(block_size), ctypes.c_float(rho), _ptr(scores), _stream(dev)))
    return scores


@_on_device
def select_start_block(scores, current_block, k_max, *, out=None):
    """Eq. (6): start block of every sequence's window.  scores: float32
    [batch, max_blocks]; current_block: int32 [batch]."""
    lib = load()
    dev = scores.device
    _need(scores, "scores", torch.float32, dev, 2)
    _need(current_block, "current_block", torch.int32, dev, 1)
    batch = current_block.shape[0]
    start = torch.empty(batch, dtype=torch.int32, device=dev) if out is None else out
    _check("mbe_select_start_block", lib.mbe_select_start_block(
        _ptr(scores), batch, scores.shape[1], _ptr(current_block), int(k_max), _ptr(start), _stream(dev)))
    return start


@_on_device
def kv_write(k_pages, v_pages, page_table, start_pos, lens, k_new, v_new, *, max_len=None, block_flags=None,
             block_size=None):
    """Write recomputed K/V (bf16 [total_tokens, heads, D]) into the paged
    pools in place: token t of sequence b goes to position start_pos[b] + t.
    The V pool's layout is read from its shape (see v_layout_of).
    block_flags: optional uint8 [batch, ceil(max_len / block_size)] device
    tensor; only tokens of flagged blocks (t // block_size) are written."""
    lib = load()
    dev = k_pages.device
    _need(k_pages, "k_pages", torch.bfloat16, dev, 4)
    _need(v_pages, "v_pages", torch.bfloat16, dev, 4)
    _need(page_table, "page_table", torch.int32, dev, 2)
    _need(start_pos, "start_pos", torch.int32, dev, 1)
    _need(lens, "lens", torch.int32, dev, 1)
    _need(k_new, "k_new", torch.bfloat16, dev, 3)
    _need(v_new, "v_new", torch.bfloat16, dev, 3)
    batch = start_pos.shape[0]
    if max_len is None:
        max_len = int(lens.max().item()) if batch else 0
    if block_flags is not None:
        if block_size is None or int(block_size) < 1:
            raise ValueError("block_flags needs block_size >= 1")
        _flags_gate(block_flags, (batch, -(-int(max_len) // int(block_size))), None, dev)
    layout = v_layout_of(k_pages, v_pages)
    _check("mbe_kv_write", lib.mbe_kv_write(
        _ptr(k_pages), _ptr(v_pages), k_pages.shape[0], k_pages.shape[1], k_pages.shape[3], layout, _ptr(page_table),
        page_table.shape[1], _ptr(start_pos), _ptr(lens), batch, int(max_len), k_new.shape[0], _ptr(k_new),
        _ptr(v_new), _ptr(block_flags), int(block_size or 0), _stream(dev)))


@_on_device
def refresh_blocks(block_changed, mode="changed", *, out=None):
    """Blocks to recompute after editing from per-block changed flags
    (uint8 [batch, num_blocks]); mode "changed" or "changed_and_later"."""
    lib = load()
    dev = block_changed.device
    _need(block_changed, "block_changed", torch.uint8, dev, 2)
    refresh = torch.empty_like(block_changed) if out is None else out
    _check("mbe_refresh_blocks", lib.mbe_refresh_blocks(
        _ptr(block_changed), block_changed.shape[0], block_changed.shape[1], REFRESH_MODES[mode], _ptr(refresh),
        _stream(dev)))
    return refresh
