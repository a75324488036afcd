"""Multi-shape HIP-graph pool for the editing pass.

Paper, Sec. "Infrastructure Optimization", multi-shape graph pool: graphs
are captured per (batch size, forward length) at start-up over a statically
allocated maximum-shape input buffer, shorter shapes use views of that
buffer, and each pass replays the graph of its shape instead of launching
eagerly.  Here one graph holds one editing pass of the library: window
attention over the paged cache followed by the full threshold update (and
the row entropies) on the pass's logits.

The caller fills the static inputs (views returned by `inputs`) and reads the
static outputs (`outputs`); `replay` runs the captured launches on the current
stream.  The attention plan is made from bounds only (`max_prefix_len`, the
shape's window), so a graph stays valid for any prefix lengths up to the
bound; the kernels read the lengths from the device buffers at run time.
Workspaces are owned per shape, so no call allocates during capture or
replay, and the captured kernels contain no memory-set operations.
"""
from __future__ import annotations

from typing import Dict, Tuple

import torch

from . import (threshold_update, window_attention, workspace_bytes_threshold_update,
               workspace_bytes_window_attention)


class EditPassGraphs:
    def __init__(self, *, k_pages, v_pages, max_batch, max_window, block_size, num_q_heads, max_pages_per_seq,
                 max_prefix_len, vocab, mask_id, omega_mask=0.5, omega_edit=0.0, with_entropy=True):
        dev = k_pages.device
        D = k_pages.shape[3]
        self.dev = dev
        self.k_pages, self.v_pages = k_pages, v_pages
        self.block_size = int(block_size)
        self.max_batch, self.max_window = int(max_batch), int(max_window)
        self.max_prefix_len = int(max_prefix_len)
        self.vocab = int(vocab)
        self.mask_id, self.omega_mask, self.omega_edit = int(mask_id), float(omega_mask), float(omega_edit)
        self.with_entropy = bool(with_entropy)
        T = self.max_batch * self.max_window
        # static maximum-shape buffers
        self.q = torch.zeros(T, num_q_heads, D, dtype=torch.bfloat16, device=dev)
        self.out = torch.zeros_like(self.q)
        self.page_table = torch.zeros(self.max_batch, max_pages_per_seq, dtype=torch.int32, device=dev)
        self.prefix_lens = torch.zeros(self.max_batch, dtype=torch.int32, device=dev)
        self.window_lens: Dict[Tuple[int, int], torch.Tensor] = {}   # per shape, filled once at capture
        self.logits = torch.zeros(T, self.vocab, dtype=torch.bfloat16, device=dev)
        self.cur = torch.zeros(T, dtype=torch.int32, device=dev)
        self.upd = {"new_tokens": torch.zeros(T, dtype=torch.int32, device=dev),
                    "conf": torch.zeros(T, dtype=torch.float32, device=dev),
                    "action": torch.zeros(T, dtype=torch.uint8, device=dev),
                    "block_changed": torch.zeros(max(T // self.block_size, 1), dtype=torch.uint8, device=dev),
                    "changed_count": torch.zeros(1, dtype=torch.int32, device=dev)}
        if self.with_entropy:
            self.upd["entropy"] = torch.zeros(T, dtype=torch.float32, device=dev)
        self.graphs: Dict[Tuple[int, int], torch.cuda.CUDAGraph] = {}
        self._ws: Dict[Tuple[int, int], Tuple[torch.Tensor, torch.Tensor]] = {}

    def _check_shape(self, batch, window):
        if not (1 <= batch <= self.max_batch and 1 <= window <= self.max_window and window % self.block_size == 0):
            raise ValueError(f"shape ({batch}, {window}) outside the pool's maximum "
                             f"({self.max_batch}, {self.max_window}) or not whole blocks")

    def inputs(self, batch, window):
        """Views of the static inputs for this shape (fill them before replay)."""
        self._check_shape(batch, window)
        n = batch * window
        return {"q": self.q[:n], "page_table": self.page_table[:batch], "prefix_lens": self.prefix_lens[:batch],
                "logits": self.logits[:n], "cur_tokens": self.cur[:n]}

    def outputs(self, batch, window):
        self._check_shape(batch, window)
        n = batch * window
        o = {"attention": self.out[:n], "changed_count": self.upd["changed_count"]}
        for k in ("new_tokens", "conf", "action") + (("entropy",) if self.with_entropy else ()):
            o[k] = self.upd[k][:n]
        o["block_changed"] = self.upd["block_changed"][: n // self.block_size]
        return o

    def _launch(self, batch, window):
        n = batch * window
        ws_attn, ws_upd = self._ws[(batch, window)]
        window_attention(self.q[:n], self.k_pages, self.v_pages, self.page_table[:batch], self.prefix_lens[:batch],
                         self.window_lens[(batch, window)], self.block_size, out=self.out[:n],
                         max_prefix_len=self.max_prefix_len, max_window_len=window, workspace=ws_attn)
        out = {k: (v[:n] if k not in ("block_changed", "changed_count") else v) for k, v in self.upd.items()}
        out["block_changed"] = self.upd["block_changed"][: n // self.block_size]
        threshold_update(self.logits[:n], self.cur[:n], self.mask_id, self.block_size, self.omega_mask,
                         self.omega_edit, with_entropy=self.with_entropy, out=out, workspace=ws_upd)

    def capture(self, batch, window):
        """Capture the pass for one shape (once; call at start-up)."""
        self._check_shape(batch, window)
        key = (batch, window)
        if key in self.graphs:
            return
        n = batch * window
        self.window_lens[key] = torch.full((batch,), window, dtype=torch.int32, device=self.dev)
        a = workspace_bytes_window_attention(self.q[:n], self.k_pages, self.page_table[:batch], batch,
                                             max_prefix_len=self.max_prefix_len, max_window_len=window)
        u = workspace_bytes_threshold_update(n, self.vocab)
        self._ws[key] = (torch.empty(max(a, 1), dtype=torch.uint8, device=self.dev),
                         torch.empty(max(u, 1), dtype=torch.uint8, device=self.dev))
        side = torch.cuda.Stream(device=self.dev)
        side.wait_stream(torch.cuda.current_stream(self.dev))
        with torch.cuda.stream(side):
            self._launch(batch, window)          # warm-up outside capture
        torch.cuda.current_stream(self.dev).wait_stream(side)
        torch.cuda.synchronize(self.dev)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self._launch(batch, window)
        self.graphs[key] = g

    def replay(self, batch, window):
        """Run the captured pass for this shape on the current stream."""
        key = (batch, window)
        g = self.graphs.get(key)
        if g is None:
            raise KeyError(f"no graph captured for shape {key}")
        g.replay()


class PassLoopGraph:
    """At most N_MBE editing passes captured as one graph, stopping early on
    the device (paper, Sec. "Training-Free MBE Decoding": at most N_MBE
    cross-block passes, stopping when no token changes).

    Pass n runs window attention over the paged cache and the full threshold
    update, in place on one token buffer.  Every pass after the first is gated
    on the previous pass's changed count (`run_if_nonzero`): once a pass
    changes nothing, the later passes' kernels exit at once, so a converged
    loop costs about a launch per remaining pass and needs no host read.

    The per-pass queries and logits are static inputs (`q[n]`, `logits[n]`):
    in a full decoder they come from the model forward on the current tokens,
    which lies outside this library.  Outputs per pass: `out[n]` (attention),
    `conf[n]`, `action[n]`, `block_changed[n]`, `counts[n]`; a gated-off pass
    leaves `out[n]` and `conf[n]` as they were and reports no change.
    """

    def __init__(self, *, k_pages, v_pages, batch, window, block_size, num_q_heads, max_pages_per_seq,
                 max_prefix_len, vocab, mask_id, n_passes=5, omega_mask=0.5, omega_edit=0.0):
        dev = k_pages.device
        D = k_pages.shape[3]
        self.dev = dev
        self.k_pages, self.v_pages = k_pages, v_pages
        self.batch, self.window, self.block_size = int(batch), int(window), int(block_size)
        if self.window % self.block_size or self.window < 1 or self.batch < 1:
            raise ValueError("window must be a positive multiple of block_size")
        self.n_passes = int(n_passes)
        self.max_prefix_len = int(max_prefix_len)
        self.vocab, self.mask_id = int(vocab), int(mask_id)
        self.omega_mask, self.omega_edit = float(omega_mask), float(omega_edit)
        T = self.batch * self.window
        n = self.n_passes
        self.q = torch.zeros(n, T, num_q_heads, D, dtype=torch.bfloat16, device=dev)
        self.out = torch.zeros_like(self.q)
        self.logits = torch.zeros(n, T, self.vocab, dtype=torch.bfloat16, device=dev)
        self.page_table = torch.zeros(self.batch, max_pages_per_seq, dtype=torch.int32, device=dev)
        self.prefix_lens = torch.zeros(self.batch, dtype=torch.int32, device=dev)
        self.window_lens = torch.full((self.batch,), self.window, dtype=torch.int32, device=dev)
        self.tokens = torch.zeros(T, dtype=torch.int32, device=dev)
        self.conf = torch.zeros(n, T, dtype=torch.float32, device=dev)
        self.action = torch.zeros(n, T, dtype=torch.uint8, device=dev)
        self.block_changed = torch.zeros(n, T // self.block_size, dtype=torch.uint8, device=dev)
        self.counts = torch.zeros(n, dtype=torch.int32, device=dev)
        a = workspace_bytes_window_attention(self.q[0], k_pages, self.page_table, self.batch,
                                             max_prefix_len=self.max_prefix_len, max_window_len=self.window)
        u = workspace_bytes_threshold_update(T, self.vocab)
        self._ws_attn = torch.empty(max(a, 1), dtype=torch.uint8, device=dev)
        self._ws_upd = torch.empty(max(u, 1), dtype=torch.uint8, device=dev)
        self.graph = None

    def _pass(self, i):
        gate = None if i == 0 else self.counts[i - 1:i]
        window_attention(self.q[i], self.k_pages, self.v_pages, self.page_table, self.prefix_lens, self.window_lens,
                         self.block_size, out=self.out[i], max_prefix_len=self.max_prefix_len,
                         max_window_len=self.window, workspace=self._ws_attn, run_if_nonzero=gate)
        out = {"new_tokens": self.tokens, "conf": self.conf[i], "action": self.action[i],
               "block_changed": self.block_changed[i], "changed_count": self.counts[i:i + 1]}
        threshold_update(self.logits[i], self.tokens, self.mask_id, self.block_size, self.omega_mask,
                         self.omega_edit, out=out, workspace=self._ws_upd, run_if_nonzero=gate)

    def run_eager(self, i):
        """Pass i alone, ungated (for host-driven loops and checks)."""
        window_attention(self.q[i], self.k_pages, self.v_pages, self.page_table, self.prefix_lens, self.window_lens,
                         self.block_size, out=self.out[i], max_prefix_len=self.max_prefix_len,
                         max_window_len=self.window, workspace=self._ws_attn)
        out = {"new_tokens": self.tokens, "conf": self.conf[i], "action": self.action[i],
               "block_changed": self.block_changed[i], "changed_count": self.counts[i:i + 1]}
        threshold_update(self.logits[i], self.tokens, self.mask_id, self.block_size, self.omega_mask,
                         self.omega_edit, out=out, workspace=self._ws_upd)

    def capture(self):
        """Capture the N_MBE gated passes (once; the static inputs may be
        refilled between replays).  Runs the passes once eagerly first (the
        warm-up), which changes `tokens`: set the tokens after capturing."""
        if self.graph is not None:
            return
        side = torch.cuda.Stream(device=self.dev)
        side.wait_stream(torch.cuda.current_stream(self.dev))
        with torch.cuda.stream(side):
            for i in range(self.n_passes):
                self._pass(i)
        torch.cuda.current_stream(self.dev).wait_stream(side)
        torch.cuda.synchronize(self.dev)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(self.n_passes):
                self._pass(i)
        self.graph = g

    def replay(self):
        if self.graph is None:
            raise RuntimeError("capture() first")
        self.graph.replay()
