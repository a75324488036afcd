"""Seeded synthetic inputs for the MBE editing-pass hot path.

This module only draws inputs: it holds none of the method's arithmetic
(no attention, no softmax, no argmax).  Both the CPU oracle (test
infrastructure) and the HIP library are fed from here, so a test compares
the two on identical bytes.

Workloads are the decoding shapes of block-diffusion MBE editing passes
(block size B = 32, window of k blocks, GQA 16/4 heads, head_dim 128,
16-token KV pages with a shuffled page table, LM-head logits over a
131072-token vocabulary).  Each is named by what it is, with its sizes.

Layouts produced (all row-major, contiguous):
  q          bf16  [total_q, num_q_heads, head_dim]       window rows of seq b
                                                          start at cu_q[b]
  k_pages    bf16  [num_pages, num_kv_heads, 16, head_dim]  token-major page
  v_pages    bf16  [num_pages, num_kv_heads, head_dim, 16]  token-minor page, or
                   [num_pages, num_kv_heads, 16, head_dim]  with v_token_major
                   (the same values, each page transposed)
  page_table int32 [batch, max_pages_per_seq]            unused slots hold 0
  prefix_lens, window_lens int32 [batch]
  logits     bf16  [rows, vocab]
  cur_tokens int32 [rows]

Random streams: numpy PCG64 keyed by (seed, case kind, tensor tag, chunk).
Attention case (kind 0): prefix lengths and the page permutation from tag 0;
Q, K, V from tags 1, 2, 3 as fp32 N(0,1) rounded to bf16 (RNE).  Edit case
(kind 1): logits from tag 1 as fp32 N(0, sigma) rounded to bf16; planted rows
and columns and current tokens from tag 0.  Large tensors are drawn in
2^22-element chunks, each from its own keyed stream, so several threads can
fill them and the values do not depend on the thread count.
"""
from __future__ import annotations

import concurrent.futures
import dataclasses
import math
import os
from typing import Optional

import numpy as np
import torch

PAGE_SIZE = 16


@dataclasses.dataclass(frozen=True)
class AttnSpec:
    batch: int
    block_size: int
    k_blocks: int            # window length in blocks (W_b = k * B)
    prefix: tuple            # ("fixed", P) or ("uniform32", lo, hi): P = 32 * U{lo..hi}
    num_q_heads: int
    num_kv_heads: int
    head_dim: int


@dataclasses.dataclass(frozen=True)
class EditSpec:
    rows: int
    vocab: int
    sigma: float
    planted_fraction: float  # fraction of rows that get one peak at max(row) + 8
    threshold: float


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    attn: AttnSpec
    edit: Optional[EditSpec]
    seed: int


# The five decoding workloads.  Seeds are fixed per workload.
WORKLOADS = {
    "tiny_p64_k2_h4_d64": Workload(
        "tiny_p64_k2_h4_d64",
        AttnSpec(1, 32, 2, ("fixed", 64), 4, 4, 64),
        EditSpec(64, 1024, 2.0, 0.0, 0.9), seed=0),
    "single_p2048_k2_gqa16x4_d128": Workload(
        "single_p2048_k2_gqa16x4_d128",
        AttnSpec(1, 32, 2, ("fixed", 2048), 16, 4, 128),
        EditSpec(64, 131072, 3.0, 0.5, 0.9), seed=1),
    "batch32_p512to8192_k2": Workload(
        "batch32_p512to8192_k2",
        AttnSpec(32, 32, 2, ("uniform32", 16, 256), 16, 4, 128),
        EditSpec(32 * 64, 131072, 3.0, 0.5, 0.9), seed=2),
    "span_sweep_b8_p16384": Workload(
        "span_sweep_b8_p16384",
        AttnSpec(8, 32, 2, ("fixed", 16384), 16, 4, 128),
        None, seed=3),
    "long_context_b64_p4096to32768_k4": Workload(
        "long_context_b64_p4096to32768_k4",
        AttnSpec(64, 32, 4, ("uniform32", 128, 1024), 16, 4, 128),
        EditSpec(64 * 128, 131072, 3.0, 0.5, 0.95), seed=4),
}

SPAN_SWEEP_K = (1, 2, 4, 8)


_CHUNK = 1 << 22
_THREADS = max(1, min(16, os.cpu_count() or 1))


def _rng(seed: int, kind: int, tag: int = 0, chunk: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64([int(seed), int(kind), int(tag), int(chunk)]))


def _normal_bf16(seed: int, kind: int, tag: int, shape, scale: float = 1.0) -> torch.Tensor:
    """N(0, scale) drawn in fp32 chunk by chunk (one keyed stream per chunk),
    rounded to bf16 (round to nearest even, by torch on the CPU)."""
    n = int(np.prod(shape))
    out = torch.empty(n, dtype=torch.bfloat16)

    def fill(i):
        s, e = i * _CHUNK, min(n, (i + 1) * _CHUNK)
        x = _rng(seed, kind, tag, i).standard_normal(e - s, dtype=np.float32)
        if scale != 1.0:
            x *= np.float32(scale)
        out[s:e] = torch.from_numpy(x).to(torch.bfloat16)

    nchunks = (n + _CHUNK - 1) // _CHUNK
    if nchunks <= 1:
        for i in range(nchunks):
            fill(i)
    else:
        with concurrent.futures.ThreadPoolExecutor(_THREADS) as ex:
            list(ex.map(fill, range(nchunks)))
    return out.view(*shape)


@dataclasses.dataclass
class AttnCase:
    q: torch.Tensor
    k_pages: torch.Tensor
    v_pages: torch.Tensor
    page_table: torch.Tensor
    prefix_lens: torch.Tensor
    window_lens: torch.Tensor
    block_size: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int

    @property
    def v_token_major(self) -> bool:
        return tuple(self.v_pages.shape[2:]) == (PAGE_SIZE, self.head_dim) and self.head_dim != PAGE_SIZE

    @property
    def batch(self) -> int:
        return int(self.prefix_lens.numel())

    @property
    def cu_q(self) -> np.ndarray:
        w = self.window_lens.numpy().astype(np.int64)
        return np.concatenate([[0], np.cumsum(w)])

    def to(self, device) -> "AttnCase":
        return dataclasses.replace(
            self, q=self.q.to(device), k_pages=self.k_pages.to(device),
            v_pages=self.v_pages.to(device), page_table=self.page_table.to(device),
            prefix_lens=self.prefix_lens.to(device), window_lens=self.window_lens.to(device))


def draw_prefix_lens(rng: np.random.Generator, spec: AttnSpec) -> np.ndarray:
    kind = spec.prefix[0]
    if kind == "fixed":
        return np.full(spec.batch, spec.prefix[1], dtype=np.int32)
    if kind == "uniform32":
        lo, hi = spec.prefix[1], spec.prefix[2]
        return (32 * rng.integers(lo, hi + 1, size=spec.batch)).astype(np.int32)
    raise ValueError(kind)


def make_attention_case(spec: AttnSpec, seed: int, *,
                        prefix_lens=None, window_lens=None,
                        q_scale: float = 1.0, extra_pages: int = 0,
                        tail_fill: Optional[float] = None, v_token_major: bool = False) -> AttnCase:
    """Draw one paged-KV attention case.

    prefix_lens / window_lens override the spec's lengths (window lengths must
    be multiples of block_size).  q_scale multiplies Q before rounding (a
    larger spread of scores).  extra_pages adds unreferenced pages to the
    pool.  tail_fill, if given, overwrites every pool slot that no sequence
    references (the tail of each sequence's last page and the extra pages)
    with that value, e.g. NaN, to show those slots are never read.
    v_token_major lays V out like K ([page, head, 16, D]) with the same values.
    """
    rng = _rng(seed, 0)
    drawn = draw_prefix_lens(rng, spec)
    P = np.asarray(drawn if prefix_lens is None else prefix_lens, dtype=np.int32)
    if window_lens is None:
        W = np.full(P.shape[0], spec.k_blocks * spec.block_size, dtype=np.int32)
    else:
        W = np.asarray(window_lens, dtype=np.int32)
    assert P.shape == W.shape
    B = spec.block_size
    Hq, Hkv, D = spec.num_q_heads, spec.num_kv_heads, spec.head_dim
    total_q = int(W.sum())
    q = _normal_bf16(seed, 0, 1, (total_q, Hq, D), scale=q_scale)
    n_tok = P.astype(np.int64) + W
    n_pages = (n_tok + PAGE_SIZE - 1) // PAGE_SIZE
    num_pages = int(n_pages.sum()) + int(extra_pages)
    k_pages = _normal_bf16(seed, 0, 2, (num_pages, Hkv, PAGE_SIZE, D))
    v_pages = _normal_bf16(seed, 0, 3, (num_pages, Hkv, D, PAGE_SIZE))
    perm = rng.permutation(num_pages).astype(np.int32)
    max_pages = max(1, int(n_pages.max()) if len(n_pages) else 1)
    page_table = np.zeros((P.shape[0], max_pages), dtype=np.int32)
    off = 0
    for b in range(P.shape[0]):
        page_table[b, :n_pages[b]] = perm[off:off + n_pages[b]]
        off += int(n_pages[b])
    if tail_fill is not None:
        used = np.zeros((num_pages, PAGE_SIZE), dtype=bool)
        for b in range(P.shape[0]):
            for t in range(int(n_tok[b])):
                used[page_table[b, t // PAGE_SIZE], t % PAGE_SIZE] = True
        unused = torch.from_numpy(~used)
        kf = k_pages.float()
        vf = v_pages.float()
        kf[unused.unsqueeze(1).unsqueeze(-1).expand_as(kf)] = tail_fill
        vf[unused.unsqueeze(1).unsqueeze(2).expand_as(vf)] = tail_fill
        k_pages = kf.to(torch.bfloat16)
        v_pages = vf.to(torch.bfloat16)
    if v_token_major:
        v_pages = v_pages.transpose(2, 3).contiguous()
    return AttnCase(q=q, k_pages=k_pages, v_pages=v_pages,
                    page_table=torch.from_numpy(page_table),
                    prefix_lens=torch.from_numpy(P.copy()),
                    window_lens=torch.from_numpy(W.copy()),
                    block_size=B, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D)


@dataclasses.dataclass
class EditCase:
    logits: torch.Tensor        # bf16 [rows, vocab]
    cur_tokens: torch.Tensor    # int32 [rows]
    threshold: float
    planted_rows: np.ndarray    # int64 row ids that received a peak
    planted_cols: np.ndarray    # int64 column of that peak


def make_edit_case(spec: EditSpec, seed: int, *, rows: Optional[int] = None,
                   cur_hit_fraction: float = 0.0) -> EditCase:
    """Draw one edit-selection case.

    Logits are fp32 N(0, sigma) rounded to bf16.  In floor(rows *
    planted_fraction) rows chosen without replacement, one uniformly chosen
    column is set to bf16(row max + 8).  Current tokens are uniform in
    [0, vocab); with cur_hit_fraction > 0 that fraction of the planted rows
    has its current token set to the planted column.
    """
    rng = _rng(seed, 1)
    R = spec.rows if rows is None else int(rows)
    V = spec.vocab
    logits = _normal_bf16(seed, 1, 1, (R, V), scale=spec.sigma)
    n_plant = int(math.floor(R * spec.planted_fraction))
    prow = np.sort(rng.choice(R, size=n_plant, replace=False)) if n_plant else np.zeros(0, np.int64)
    pcol = rng.integers(0, V, size=n_plant)
    if n_plant:
        rmax = logits[torch.from_numpy(prow)].float().amax(dim=1)
        logits[torch.from_numpy(prow), torch.from_numpy(pcol)] = (rmax + 8.0).to(torch.bfloat16)
    cur = rng.integers(0, V, size=R).astype(np.int32)
    if cur_hit_fraction > 0 and n_plant:
        nh = int(n_plant * cur_hit_fraction)
        hit = rng.choice(n_plant, size=nh, replace=False)
        cur[prow[hit]] = pcol[hit]
    return EditCase(logits=logits, cur_tokens=torch.from_numpy(cur),
                    threshold=float(spec.threshold),
                    planted_rows=prow.astype(np.int64), planted_cols=pcol.astype(np.int64))


def workload_attention(name: str, k_blocks: Optional[int] = None, **kw) -> AttnCase:
    w = WORKLOADS[name]
    spec = w.attn if k_blocks is None else dataclasses.replace(w.attn, k_blocks=int(k_blocks))
    return make_attention_case(spec, w.seed, **kw)


def workload_edit(name: str, **kw) -> EditCase:
    w = WORKLOADS[name]
    assert w.edit is not None, f"{name} has no edit-selection step"
    return make_edit_case(w.edit, w.seed, **kw)
