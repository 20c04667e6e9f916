"""Seeded synthetic inputs for paged rollout attention.

Shared by the tests, the benchmark and the smoke check: it feeds both the HIP
library and the CPU oracle, so it holds none of the attention arithmetic. It
only draws lengths, lays trajectories out on shuffled physical pages, and fills
pools and queries with bf16 N(0, 1) values.

Workload shapes follow the multi-turn agent rollouts of the ProRL Agent paper:
a single agent trajectory can run for many tens of turns and grow to many
thousands of tokens, into the tens of thousands (Sec. 1); every agent step
decodes over the whole history kept so far (Sec. 3.3.2); and the output of a
tool or of the environment is added after the tokens already kept
(Sec. 3.3.3).

Recipe (every choice the workload descriptions leave open is stated here):
  * lengths and page permutations: numpy.random.default_rng(seed);
    "uniform in [a, b]" is the discrete uniform over integers, both ends in;
    "log-normal with median m" is round(exp(N(ln m, 0.75))) clipped to the range;
  * pages: each row needs ceil(len / 16) pages; the pool has those pages plus
    max(16, 1 %) decoy pages; physical ids come from one random permutation;
    block-table entries past a row's last page point at decoy pages;
  * values: torch.Generator seeded with 1000 + seed on the target device,
    fp32 N(0, 1) rounded to bf16 (round to nearest even), drawn in the order
    K pool, V pool, queries, new keys, new values.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np
import torch

PAGE = 16
HEAD_DIM = 128
BF16_NAN = 0x7FC0


@dataclasses.dataclass
class PagedLayout:
    """Rows laid out on shuffled pages. Lengths are in tokens."""
    num_pages: int
    block_table: np.ndarray      # int32 [B][stride]
    row_tokens: np.ndarray       # int32 [B], tokens resident in the cache per row
    decoys: np.ndarray           # int32, page ids no row owns


@dataclasses.dataclass
class Workload:
    """One batch of rollout attention work over a shared pool."""
    name: str
    Hq: int
    Hkv: int
    layout: PagedLayout
    # decode rows (indices into the layout's rows) and their key counts
    decode_rows: np.ndarray      # int32 [Bd]
    kv_lens: np.ndarray          # int32 [Bd]
    # append rows, their cached context and chunk length
    append_rows: np.ndarray      # int32 [Ba]
    ctx_lens: np.ndarray         # int32 [Ba]
    q_lens: np.ndarray           # int32 [Ba]
    seed: int
    head_dim: int = HEAD_DIM
    page_size: int = PAGE
    # shared-prefix decode: row offsets of the groups [G + 1] and the tokens
    # the rows of each group share [G] (None for other workloads)
    group_start: Optional[np.ndarray] = None
    prefix_len: Optional[np.ndarray] = None

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    def decode_table(self) -> np.ndarray:
        return np.ascontiguousarray(self.layout.block_table[self.decode_rows])

    def append_table(self) -> np.ndarray:
        return np.ascontiguousarray(self.layout.block_table[self.append_rows])

    def cu_q(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.q_lens)]).astype(np.int32)


def uniform_int(rng: np.random.Generator, n: int, lo: int, hi: int) -> np.ndarray:
    return rng.integers(lo, hi + 1, size=n).astype(np.int64)


def lognormal_int(rng: np.random.Generator, n: int, median: float, sigma: float, lo: int,
                  hi: int) -> np.ndarray:
    x = np.rint(np.exp(rng.normal(math.log(median), sigma, size=n)))
    return np.clip(x, lo, hi).astype(np.int64)


def make_layout(rng: np.random.Generator, row_tokens, page_size: int = PAGE,
                decoy_frac: float = 0.01, min_decoys: int = 16,
                extra_stride: int = 0) -> PagedLayout:
    row_tokens = np.asarray(row_tokens, dtype=np.int64)
    pages = (row_tokens + page_size - 1) // page_size
    n_used = int(pages.sum())
    n_decoy = max(min_decoys, int(math.ceil(decoy_frac * n_used)))
    num_pages = n_used + n_decoy
    perm = rng.permutation(num_pages).astype(np.int32)
    decoys = perm[n_used:]
    stride = max(1, int(pages.max()) if pages.size else 1) + extra_stride
    B = row_tokens.shape[0]
    bt = np.empty((B, stride), np.int32)
    off = 0
    for b in range(B):
        n = int(pages[b])
        bt[b, :n] = perm[off:off + n]
        rest = stride - n
        if rest:
            bt[b, n:] = decoys[(b + np.arange(rest)) % n_decoy]
        off += n
    return PagedLayout(num_pages, bt, row_tokens.astype(np.int32), decoys)


def shared_prefix_layout(rng: np.random.Generator, group_sizes, prefix_tokens, suffix_tokens,
                         page_size: int = PAGE, decoy_frac: float = 0.01,
                         min_decoys: int = 16) -> PagedLayout:
    """Rows in consecutive groups; the rows of group i share the pages of their
    first prefix_tokens[i] tokens (a multiple of the page size), then each row
    owns the pages of its suffix_tokens[r] further tokens. Page ids shuffled."""
    sizes = np.asarray(group_sizes, np.int64)
    pre = np.asarray(prefix_tokens, np.int64)
    suf = np.asarray(suffix_tokens, np.int64)
    assert np.all(pre % page_size == 0) and suf.shape[0] == sizes.sum()
    row_group = np.repeat(np.arange(sizes.shape[0]), sizes)
    pre_pages = pre // page_size
    suf_pages = (suf + page_size - 1) // page_size
    n_used = int(pre_pages.sum() + suf_pages.sum())
    n_decoy = max(min_decoys, int(math.ceil(decoy_frac * n_used)))
    num_pages = n_used + n_decoy
    perm = rng.permutation(num_pages).astype(np.int32)
    decoys = perm[n_used:]
    row_pages = pre_pages[row_group] + suf_pages
    stride = max(1, int(row_pages.max()))
    B = suf.shape[0]
    bt = np.empty((B, stride), np.int32)
    off = 0
    shared = []
    for i in range(sizes.shape[0]):
        shared.append(perm[off:off + int(pre_pages[i])])
        off += int(pre_pages[i])
    for b in range(B):
        sp = shared[row_group[b]]
        n = int(suf_pages[b])
        bt[b, :sp.shape[0]] = sp
        bt[b, sp.shape[0]:sp.shape[0] + n] = perm[off:off + n]
        rest = stride - sp.shape[0] - n
        if rest:
            bt[b, stride - rest:] = decoys[(b + np.arange(rest)) % n_decoy]
        off += n
    return PagedLayout(num_pages, bt, (pre[row_group] + suf).astype(np.int32), decoys)


def shared_prefix_workload(seed: int, n_groups: int, rows_per_group: int, Hq: int, Hkv: int,
                           prefix, suffix, name: str) -> Workload:
    """Decode rows in groups of rows_per_group that share a prefix (whole pages)."""
    rng = np.random.default_rng(seed)
    pre = np.asarray(prefix(rng, n_groups), np.int64) // PAGE * PAGE
    B = n_groups * rows_per_group
    suf = np.asarray(suffix(rng, B), np.int64)
    lay = shared_prefix_layout(rng, [rows_per_group] * n_groups, pre, suf)
    e = np.zeros(0, np.int32)
    gs = (np.arange(n_groups + 1) * rows_per_group).astype(np.int32)
    return Workload(name, Hq, Hkv, lay, np.arange(B, dtype=np.int32),
                    lay.row_tokens.astype(np.int32), e, e, e, seed,
                    group_start=gs, prefix_len=pre.astype(np.int32))


# ---------------------------------------------------------------------------
# The five rollout workloads (lengths in tokens, page size 16, head dim 128).
# ---------------------------------------------------------------------------

def decode_workload(seed: int, B: int, Hq: int, Hkv: int, lens, name: str) -> Workload:
    rng = np.random.default_rng(seed)
    lens = np.asarray(lens(rng, B), np.int64)
    lay = make_layout(rng, lens)
    e = np.zeros(0, np.int32)
    return Workload(name, Hq, Hkv, lay, np.arange(B, dtype=np.int32), lens.astype(np.int32),
                    e, e, e, seed)


def append_workload(seed: int, B: int, Hq: int, Hkv: int, ctx, qlen, name: str) -> Workload:
    rng = np.random.default_rng(seed)
    c = np.asarray(ctx(rng, B), np.int64)
    t = np.asarray(qlen(rng, B), np.int64)
    lay = make_layout(rng, c + t)
    e = np.zeros(0, np.int32)
    return Workload(name, Hq, Hkv, lay, e, e, np.arange(B, dtype=np.int32),
                    c.astype(np.int32), t.astype(np.int32), seed)


def mixed_workload(seed: int, B: int, Hq: int, Hkv: int, append_frac: float, ctx, qlen,
                   name: str) -> Workload:
    rng = np.random.default_rng(seed)
    n_app = int(round(append_frac * B))
    is_app = np.zeros(B, bool)
    is_app[rng.permutation(B)[:n_app]] = True
    c = np.asarray(ctx(rng, B), np.int64)
    t = np.where(is_app, np.asarray(qlen(rng, B), np.int64), 0)
    lay = make_layout(rng, c + t)
    dec = np.nonzero(~is_app)[0].astype(np.int32)
    app = np.nonzero(is_app)[0].astype(np.int32)
    return Workload(name, Hq, Hkv, lay, dec, c[dec].astype(np.int32), app,
                    c[app].astype(np.int32), t[app].astype(np.int32), seed)


def config(c: int) -> Workload:
    """The rollout-attention workloads, numbered 1..6 (6: shared-prefix decode)."""
    if c == 1:
        return decode_workload(1, 4, 8, 2, lambda r, n: uniform_int(r, n, 32, 256),
                               "decode B=4 Hq=8 Hkv=2 L~U[32,256]")
    if c == 2:
        return decode_workload(2, 64, 32, 8, lambda r, n: uniform_int(r, n, 4096, 32768),
                               "decode Qwen3-8B GQA B=64 Hq=32 Hkv=8 L~U[4096,32768]")
    if c == 3:
        return append_workload(3, 32, 32, 8, lambda r, n: uniform_int(r, n, 2048, 24576),
                               lambda r, n: uniform_int(r, n, 64, 2048),
                               "append Qwen3-8B GQA B=32 Hq=32 Hkv=8 ctx~U[2048,24576] "
                               "T~U[64,2048]")
    if c == 4:
        return decode_workload(4, 256, 64, 8,
                               lambda r, n: lognormal_int(r, n, 16384, 0.75, 512, 65536),
                               "decode 32B-like B=256 Hq=64 Hkv=8 L~LN(16384,0.75)"
                               "[512,65536]")
    if c == 5:
        return mixed_workload(5, 512, 32, 8, 0.15,
                              lambda r, n: lognormal_int(r, n, 12288, 0.75, 512, 65536),
                              lambda r, n: uniform_int(r, n, 128, 4096),
                              "mixed B=512 Hq=32 Hkv=8 85% decode / 15% append "
                              "ctx~LN(12288,0.75)[512,65536] T~U[128,4096]")
    if c == 6:
        return shared_prefix_workload(6, 8, 8, 32, 8,
                                      lambda r, n: uniform_int(r, n, 2048, 8192),
                                      lambda r, n: uniform_int(r, n, 2048, 24576),
                                      "decode shared prefix B=64 (8 tasks x 8 rollouts) "
                                      "Hq=32 Hkv=8 prompt~U[2048,8192] "
                                      "rollout~U[2048,24576]")
    raise ValueError(f"unknown workload {c}")


# ---------------------------------------------------------------------------
# Values
# ---------------------------------------------------------------------------

def value_generator(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(1000 + seed)
    return g


def randn_bf16(shape, gen: torch.Generator, device, chunk: int = 1 << 28) -> torch.Tensor:
    """bf16 N(0,1) tensor, drawn in fp32 chunks and rounded to nearest even."""
    out = torch.empty(shape, dtype=torch.bfloat16, device=device)
    flat = out.view(-1)
    n = flat.numel()
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        flat[s:e] = torch.randn(e - s, generator=gen, device=device,
                                dtype=torch.float32).to(torch.bfloat16)
    return out


def randn_fp8_codes(shape, gen: torch.Generator, device, scale: float,
                    chunk: int = 1 << 28) -> torch.Tensor:
    """E4M3 codes (uint8) of N(0,1) values stored with the given pool scale: N(0,1) / scale
    clamped to +-448 and rounded to E4M3 by torch (round to nearest even)."""
    out = torch.empty(shape, dtype=torch.uint8, device=device)
    flat = out.view(-1)
    n = flat.numel()
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        x = torch.randn(e - s, generator=gen, device=device, dtype=torch.float32) / scale
        flat[s:e] = x.clamp(-448.0, 448.0).to(torch.float8_e4m3fn).view(torch.uint8)
    return out


@dataclasses.dataclass
class Tensors:
    k_pool: torch.Tensor     # bf16 [pages][Hkv][16][128]
    v_pool: torch.Tensor     # bf16 [pages][Hkv][128][16]
    q_decode: torch.Tensor   # bf16 [Bd][Hq][128]
    q_append: torch.Tensor   # bf16 [sum T][Hq][128]
    k_new: torch.Tensor      # bf16 [N_new][Hkv][128]: decode tokens then append chunks
    v_new: torch.Tensor


def make_tensors(w: Workload, device, gen: Optional[torch.Generator] = None) -> Tensors:
    gen = gen if gen is not None else value_generator(w.seed, device)
    P, D = w.page_size, w.head_dim
    n = w.layout.num_pages
    k_pool = randn_bf16((n, w.Hkv, P, D), gen, device)
    v_pool = randn_bf16((n, w.Hkv, D, P), gen, device)
    q_dec = randn_bf16((w.decode_rows.shape[0], w.Hq, D), gen, device)
    q_app = randn_bf16((int(w.q_lens.sum()), w.Hq, D), gen, device)
    n_new = w.decode_rows.shape[0] + int(w.q_lens.sum())
    k_new = randn_bf16((n_new, w.Hkv, D), gen, device)
    v_new = randn_bf16((n_new, w.Hkv, D), gen, device)
    return Tensors(k_pool, v_pool, q_dec, q_app, k_new, v_new)


def write_plan(w: Workload):
    """Rows, start positions and packed offsets of one step's new tokens.

    Decode rows write their current token at position kv_len - 1; append rows
    write their chunk at positions ctx .. ctx + T - 1. Returns (block_table,
    cu_new, start_pos) over the decode rows followed by the append rows.
    """
    rows = np.concatenate([w.decode_rows, w.append_rows]).astype(np.int64)
    counts = np.concatenate([np.ones(w.decode_rows.shape[0], np.int64),
                             w.q_lens.astype(np.int64)])
    start = np.concatenate([w.kv_lens.astype(np.int64) - 1, w.ctx_lens.astype(np.int64)])
    cu = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    bt = np.ascontiguousarray(w.layout.block_table[rows])
    return bt, cu, start.astype(np.int32)


def poison_unowned(k_pool: torch.Tensor, v_pool: torch.Tensor, layout: PagedLayout,
                   rows=None, lens=None) -> None:
    """Fill decoy pages and every slot past each row's length with NaN (in place).

    rows/lens: the rows whose tail slots to poison and their lengths in tokens
    (defaults: every row, its resident token count).
    """
    P = k_pool.shape[2]
    if k_pool.dtype == torch.uint8:      # fp8 pools: the E4M3 NaN code
        nan = 0x7F
    else:
        nan = torch.tensor(BF16_NAN, dtype=torch.int16).view(torch.bfloat16).item()
    dec = torch.as_tensor(layout.decoys.astype(np.int64), device=k_pool.device)
    k_pool[dec] = nan
    v_pool[dec] = nan
    rows = np.arange(layout.block_table.shape[0]) if rows is None else np.asarray(rows)
    lens = layout.row_tokens[rows] if lens is None else np.asarray(lens)
    for r, L in zip(rows.tolist(), lens.tolist()):
        if L % P:
            page = int(layout.block_table[r, L // P])
            k_pool[page, :, L % P:, :] = nan
            v_pool[page, :, :, L % P:] = nan


# ---------------------------------------------------------------------------
# Host copies (for the CPU oracle): bit patterns and the pages of a few rows
# ---------------------------------------------------------------------------

def bits(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor (any device) -> host uint16 bit patterns; a uint8 tensor (E4M3
    codes of an fp8 pool) -> host uint8."""
    t = t.detach().contiguous()
    if t.dtype == torch.uint8:
        return t.cpu().numpy()
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def compact_rows(k_pool: torch.Tensor, v_pool: torch.Tensor, table: np.ndarray, lens):
    """Host copy of only the pages the given rows use, with a remapped block table.

    table: [R][stride] block-table rows; lens: tokens used per row. The copy is
    made with torch indexing.
    """
    P = k_pool.shape[2]
    pages = [table[r, :(int(L) + P - 1) // P] for r, L in enumerate(lens)]
    ids = np.unique(np.concatenate(pages)) if pages else np.zeros(0, np.int64)
    idx = torch.as_tensor(ids.astype(np.int64), device=k_pool.device)
    k = bits(k_pool.index_select(0, idx))
    v = bits(v_pool.index_select(0, idx))
    remap = {int(p): i for i, p in enumerate(ids)}
    stride = max(1, max(len(p) for p in pages)) if pages else 1
    bt = np.zeros((len(pages), stride), np.int32)
    for r, p in enumerate(pages):
        bt[r, :len(p)] = [remap[int(x)] for x in p]
    return k, v, bt
