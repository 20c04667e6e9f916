"""MI355X rollout attention: paged-KV decode, observation append and page writes.

Thin PyTorch-facing binding of the C ABI in include/rollout_attn.h. It only
checks tensor dtypes/devices, allocates outputs with torch and passes raw
device pointers plus torch's current HIP stream to the library; every step of
the computation runs in the library's HIP kernels. If the library is not built
the import of any function fails loudly: there is no fallback path.

Host-side sizes (max_kv_len, max_q_len, max_new, max_pos, total, ...) that are
left as None are read from the device tensors with .item(), which waits for the
GPU: such a call is neither asynchronous nor capturable into a HIP graph. Pass
them explicitly (and an output and workspace) to capture a call or to keep it
asynchronous. With stream= given, outputs and workspaces the wrapper allocates
are recorded on that stream, so torch does not reuse their memory before the
call's kernels finish.

Layout (see the header): K pool [pages][Hkv][16][128] (token-major), V pool
[pages][Hkv][128][16] (dim-major), block table int32 [B][stride]. Pools are
bf16, or uint8 OCP FP8 E4M3 codes with one scale per pool (value = code * scale).
"""
from __future__ import annotations

import ctypes
import math
from typing import Optional, Tuple

import torch

from . import _lib
from ._lib import RolloutAttnError  # noqa: F401  (re-export)

PAGE_SIZE = 16
HEAD_DIM = 128

__all__ = ["PagedKV", "decode", "decode_noalloc", "decode_shared_prefix", "append", "append_write", "mixed",
           "kv_page_write",
           "kv_page_gather", "token_logprob", "decode_workspace_size",
           "decode_shared_prefix_workspace_size", "append_workspace_size", "mixed_workspace_size",
           "token_logprob_workspace_size", "token_logprob_pack_weight", "token_logprob_packed",
           "abi_version", "RolloutAttnError"]


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _need(t: torch.Tensor, name: str, dtype: torch.dtype, device: torch.device) -> None:
    # the kernels dereference every pointer on the GPU: host tensors are refused
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor, got one on {t.device}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.device != device:
        raise ValueError(f"{name} must be on {device}, got {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _shape(t: torch.Tensor, shape, name: str) -> None:
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def _rows(kv: "PagedKV", B: int) -> None:
    if kv.block_table.shape[0] < B:
        raise ValueError(f"block_table has {kv.block_table.shape[0]} rows, batch has {B}")


def _stream(device: torch.device, stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _empty(shape, dtype: torch.dtype, device: torch.device, stream) -> torch.Tensor:
    """torch.empty for an output or workspace of a call launched on `stream`.

    torch's caching allocator ties a block to the stream that was current when it
    was allocated. When the call runs on another stream (stream= given), the block
    is also recorded on that stream, so that it is not handed to new work before
    the call's kernels are done with it (a workspace the wrapper drops on return
    would otherwise be reusable at once by work on the current stream)."""
    t = torch.empty(shape, dtype=dtype, device=device)
    if stream is not None:
        s = stream if isinstance(stream, torch.cuda.Stream) else \
            torch.cuda.ExternalStream(int(stream), device=device)
        if s.cuda_stream != torch.cuda.current_stream(device).cuda_stream:
            t.record_stream(s)
    return t


class PagedKV:
    """A caller-owned paged KV cache: two pools and a block table, all on one GPU.

    bf16 pools, or fp8 pools (torch.uint8 or torch.float8_e4m3fn storage of E4M3
    codes) with k_scale / v_scale: an element's value is code * scale.
    """

    def __init__(self, k_pool: torch.Tensor, v_pool: torch.Tensor, block_table: torch.Tensor,
                 k_scale: Optional[float] = None, v_scale: Optional[float] = None):
        dev = k_pool.device
        if k_pool.dtype == torch.float8_e4m3fn:
            k_pool = k_pool.view(torch.uint8)
        if v_pool.dtype == torch.float8_e4m3fn:
            v_pool = v_pool.view(torch.uint8)
        self.fp8 = k_pool.dtype == torch.uint8
        dt = torch.uint8 if self.fp8 else torch.bfloat16
        _need(k_pool, "k_pool", dt, dev)
        _need(v_pool, "v_pool", dt, dev)
        if self.fp8 and (k_scale is None or v_scale is None):
            raise ValueError("fp8 pools need k_scale and v_scale")
        self.k_scale = float(k_scale) if self.fp8 else 1.0
        self.v_scale = float(v_scale) if self.fp8 else 1.0
        _need(block_table, "block_table", torch.int32, dev)
        if k_pool.dim() != 4 or k_pool.shape[2:] != (PAGE_SIZE, HEAD_DIM):
            raise ValueError(f"k_pool must be [pages][Hkv][16][128], got {tuple(k_pool.shape)}")
        n, hkv = k_pool.shape[:2]
        if tuple(v_pool.shape) != (n, hkv, HEAD_DIM, PAGE_SIZE):
            raise ValueError(f"v_pool must be [pages][Hkv][128][16], got {tuple(v_pool.shape)}")
        if block_table.dim() != 2:
            raise ValueError("block_table must be [B][stride]")
        self.k_pool, self.v_pool, self.block_table = k_pool, v_pool, block_table
        self.device = dev
        self.num_pages, self.num_kv_heads = int(n), int(hkv)
        self.bt_stride = int(block_table.shape[1])

    def with_table(self, block_table: torch.Tensor) -> "PagedKV":
        """Same pools, another block table (e.g. a sub-batch of rows)."""
        return PagedKV(self.k_pool, self.v_pool, block_table,
                       self.k_scale if self.fp8 else None, self.v_scale if self.fp8 else None)

    def struct(self) -> _lib.RaPagedKV:
        return _lib.RaPagedKV(self.k_pool.data_ptr(), self.v_pool.data_ptr(),
                              self.block_table.data_ptr(), self.num_pages, self.bt_stride,
                              self.num_kv_heads, PAGE_SIZE, HEAD_DIM,
                              _lib.RA_KV_FP8_E4M3 if self.fp8 else _lib.RA_KV_BF16,
                              self.k_scale, self.v_scale)


def abi_version() -> int:
    return _lib.load().ra_abi_version()


def decode_workspace_size(B: int, Hq: int, Hkv: int, max_kv_len: int) -> int:
    return int(_lib.load().rollout_attn_decode_workspace_size(B, Hq, Hkv, max_kv_len))


def decode(q: torch.Tensor, kv: PagedKV, kv_lens: torch.Tensor, max_kv_len: Optional[int] = None,
           scale: Optional[float] = None, out: Optional[torch.Tensor] = None,
           lse: Optional[torch.Tensor] = None, want_lse: bool = False,
           workspace: Optional[torch.Tensor] = None, stream=None
           ) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """Decode attention; q bf16 [B][Hq][128] -> out fp32 [B][Hq][128] (, lse fp32 [B][Hq])."""
    lib = _lib.load()
    dev = kv.device
    _need(q, "q", torch.bfloat16, dev)
    _need(kv_lens, "kv_lens", torch.int32, dev)
    B, Hq, D = q.shape
    _shape(q, (B, Hq, HEAD_DIM), "q")
    _shape(kv_lens, (B,), "kv_lens")
    _rows(kv, B)
    if max_kv_len is None:
        max_kv_len = int(kv_lens.max().item()) if B else 0
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if out is None:
        out = _empty((B, Hq, D), torch.float32, dev, stream)
    _need(out, "out", torch.float32, dev)
    _shape(out, (B, Hq, HEAD_DIM), "out")
    if lse is None and want_lse:
        lse = _empty((B, Hq), torch.float32, dev, stream)
    if lse is not None:
        _need(lse, "lse", torch.float32, dev)
        _shape(lse, (B, Hq), "lse")
    ws_bytes = lib.rollout_attn_decode_workspace_size(B, Hq, kv.num_kv_heads, max_kv_len)
    if workspace is None:
        workspace = _empty(max(ws_bytes, 1), torch.uint8, dev, stream)
    _need(workspace, "workspace", torch.uint8, dev)
    s = kv.struct()
    _lib.check("rollout_attn_decode", lib.rollout_attn_decode(
        q.data_ptr(), ctypes.byref(s), kv_lens.data_ptr(), B, Hq, max_kv_len, float(scale),
        out.data_ptr(), _ptr(lse), workspace.data_ptr(), workspace.numel(), _stream(dev, stream)))
    return out, lse


def decode_noalloc(q: torch.Tensor, kv: PagedKV, kv_lens: torch.Tensor, max_kv_len: int,
                   out: torch.Tensor, scale: Optional[float] = None,
                   lse: Optional[torch.Tensor] = None, stream=None
                   ) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """decode() without a workspace: the library's own per-GPU device scratch holds
    the split partials, so the call allocates nothing (the caller passes out, and
    lse if wanted, and the host-side max_kv_len). Plans needing more than
    RA_NOALLOC_SCRATCH_BYTES of partials are refused (RA_ERR_WORKSPACE). Calls
    that overlap on one GPU share that scratch and race: keep them on one stream."""
    lib = _lib.load()
    dev = kv.device
    _need(q, "q", torch.bfloat16, dev)
    _need(kv_lens, "kv_lens", torch.int32, dev)
    B, Hq, D = q.shape
    _shape(q, (B, Hq, HEAD_DIM), "q")
    _shape(kv_lens, (B,), "kv_lens")
    _rows(kv, B)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    _need(out, "out", torch.float32, dev)
    _shape(out, (B, Hq, HEAD_DIM), "out")
    if lse is not None:
        _need(lse, "lse", torch.float32, dev)
        _shape(lse, (B, Hq), "lse")
    s = kv.struct()
    _lib.check("rollout_attn_decode_noalloc", lib.rollout_attn_decode_noalloc(
        q.data_ptr(), ctypes.byref(s), kv_lens.data_ptr(), B, Hq, int(max_kv_len), float(scale),
        out.data_ptr(), _ptr(lse), _stream(dev, stream)))
    return out, lse


def decode_shared_prefix_workspace_size(B: int, Hq: int, Hkv: int, max_kv_len: int,
                                        max_prefix_len: int) -> int:
    return int(_lib.load().rollout_attn_decode_shared_prefix_workspace_size(
        B, Hq, Hkv, max_kv_len, max_prefix_len))


def decode_shared_prefix(q: torch.Tensor, kv: PagedKV, kv_lens: torch.Tensor,
                         group_start: torch.Tensor, prefix_len: torch.Tensor,
                         max_group_rows: int, max_prefix_len: int,
                         max_kv_len: Optional[int] = None, scale: Optional[float] = None,
                         out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                         want_lse: bool = False, workspace: Optional[torch.Tensor] = None,
                         stream=None) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """Decode for groups of rows that share their first prefix_len[i] cached tokens.

    group_start int32 [G+1] (row offsets of the groups), prefix_len int32 [G];
    the result equals decode() on the same rows up to rounding.
    """
    lib = _lib.load()
    dev = kv.device
    _need(q, "q", torch.bfloat16, dev)
    _need(kv_lens, "kv_lens", torch.int32, dev)
    _need(group_start, "group_start", torch.int32, dev)
    _need(prefix_len, "prefix_len", torch.int32, dev)
    B, Hq, D = q.shape
    _shape(q, (B, Hq, HEAD_DIM), "q")
    _shape(kv_lens, (B,), "kv_lens")
    ng = prefix_len.shape[0]
    _shape(group_start, (ng + 1,), "group_start")
    _rows(kv, B)
    if max_kv_len is None:
        max_kv_len = int(kv_lens.max().item()) if B else 0
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if out is None:
        out = _empty((B, Hq, D), torch.float32, dev, stream)
    _need(out, "out", torch.float32, dev)
    _shape(out, (B, Hq, HEAD_DIM), "out")
    if lse is None and want_lse:
        lse = _empty((B, Hq), torch.float32, dev, stream)
    if lse is not None:
        _need(lse, "lse", torch.float32, dev)
        _shape(lse, (B, Hq), "lse")
    ws_bytes = lib.rollout_attn_decode_shared_prefix_workspace_size(
        B, Hq, kv.num_kv_heads, max_kv_len, max_prefix_len)
    if workspace is None:
        workspace = _empty(max(ws_bytes, 1), torch.uint8, dev, stream)
    _need(workspace, "workspace", torch.uint8, dev)
    s = kv.struct()
    _lib.check("rollout_attn_decode_shared_prefix", lib.rollout_attn_decode_shared_prefix(
        q.data_ptr(), ctypes.byref(s), kv_lens.data_ptr(), group_start.data_ptr(),
        prefix_len.data_ptr(), B, Hq, ng, max_group_rows, max_prefix_len, max_kv_len,
        float(scale), out.data_ptr(), _ptr(lse), workspace.data_ptr(), workspace.numel(),
        _stream(dev, stream)))
    return out, lse


def append(q: torch.Tensor, cu_q: torch.Tensor, ctx_lens: torch.Tensor, kv: PagedKV,
           max_q_len: Optional[int] = None, max_kv_len: Optional[int] = None,
           scale: Optional[float] = None, out: Optional[torch.Tensor] = None,
           lse: Optional[torch.Tensor] = None, want_lse: bool = False,
           workspace: Optional[torch.Tensor] = None, stream=None
           ) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """Append attention; q bf16 [total_q][Hq][128] -> out fp32 [total_q][Hq][128]."""
    lib = _lib.load()
    dev = kv.device
    _need(q, "q", torch.bfloat16, dev)
    _need(cu_q, "cu_q", torch.int32, dev)
    _need(ctx_lens, "ctx_lens", torch.int32, dev)
    total_q, Hq, D = q.shape
    _shape(q, (total_q, Hq, HEAD_DIM), "q")
    B = ctx_lens.shape[0]
    _shape(cu_q, (B + 1,), "cu_q")
    _rows(kv, B)
    if max_q_len is None or max_kv_len is None:
        t = (cu_q[1:] - cu_q[:-1]) if B else cu_q[:0]
        if max_q_len is None:
            max_q_len = int(t.max().item()) if B else 0
        if max_kv_len is None:
            max_kv_len = int((t + ctx_lens).max().item()) if B else 0
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if out is None:
        out = _empty((total_q, Hq, D), torch.float32, dev, stream)
    _need(out, "out", torch.float32, dev)
    _shape(out, (total_q, Hq, HEAD_DIM), "out")
    if lse is None and want_lse:
        lse = _empty((total_q, Hq), torch.float32, dev, stream)
    if lse is not None:
        _need(lse, "lse", torch.float32, dev)
        _shape(lse, (total_q, Hq), "lse")
    ws_bytes = lib.rollout_attn_append_workspace_size(B, Hq, kv.num_kv_heads, max_q_len)
    if workspace is None:
        workspace = _empty(max(ws_bytes, 1), torch.uint8, dev, stream)
    _need(workspace, "workspace", torch.uint8, dev)
    s = kv.struct()
    _lib.check("rollout_attn_append", lib.rollout_attn_append(
        q.data_ptr(), cu_q.data_ptr(), ctx_lens.data_ptr(), ctypes.byref(s), B, Hq, total_q,
        max_q_len, max_kv_len, float(scale), out.data_ptr(), _ptr(lse), workspace.data_ptr(),
        workspace.numel(), _stream(dev, stream)))
    return out, lse


def append_write(q: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor, cu_q: torch.Tensor,
                 ctx_lens: torch.Tensor, kv: PagedKV, max_q_len: Optional[int] = None,
                 max_kv_len: Optional[int] = None, scale: Optional[float] = None,
                 out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                 want_lse: bool = False, workspace: Optional[torch.Tensor] = None, stream=None,
                 cos_sin: Optional[torch.Tensor] = None
                 ) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """Write the chunks' K/V (bf16 [total_q][Hkv][128], packed like q) at positions
    ctx_lens[b] + i and run the append attention, in one launch. With a rotary table
    cos_sin (fp32 [rows][128]) the chunk's keys and queries are rotated at their
    positions."""
    lib = _lib.load()
    dev = kv.device
    for t, n in ((q, "q"), (k_new, "k_new"), (v_new, "v_new")):
        _need(t, n, torch.bfloat16, dev)
    _need(cu_q, "cu_q", torch.int32, dev)
    _need(ctx_lens, "ctx_lens", torch.int32, dev)
    total_q, Hq, D = q.shape
    _shape(q, (total_q, Hq, HEAD_DIM), "q")
    _shape(k_new, (total_q, kv.num_kv_heads, HEAD_DIM), "k_new")
    _shape(v_new, (total_q, kv.num_kv_heads, HEAD_DIM), "v_new")
    B = ctx_lens.shape[0]
    _shape(cu_q, (B + 1,), "cu_q")
    _rows(kv, B)
    if max_q_len is None or max_kv_len is None:
        t = (cu_q[1:] - cu_q[:-1]) if B else cu_q[:0]
        if max_q_len is None:
            max_q_len = int(t.max().item()) if B else 0
        if max_kv_len is None:
            max_kv_len = int((t + ctx_lens).max().item()) if B else 0
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if out is None:
        out = _empty((total_q, Hq, D), torch.float32, dev, stream)
    _need(out, "out", torch.float32, dev)
    _shape(out, (total_q, Hq, HEAD_DIM), "out")
    if lse is None and want_lse:
        lse = _empty((total_q, Hq), torch.float32, dev, stream)
    if lse is not None:
        _need(lse, "lse", torch.float32, dev)
        _shape(lse, (total_q, Hq), "lse")
    ws_bytes = lib.rollout_attn_append_workspace_size(B, Hq, kv.num_kv_heads, max_q_len)
    if workspace is None:
        workspace = _empty(max(ws_bytes, 1), torch.uint8, dev, stream)
    _need(workspace, "workspace", torch.uint8, dev)
    s = kv.struct()
    if cos_sin is None:
        _lib.check("rollout_attn_append_write", lib.rollout_attn_append_write(
            q.data_ptr(), k_new.data_ptr(), v_new.data_ptr(), cu_q.data_ptr(),
            ctx_lens.data_ptr(), ctypes.byref(s), B, Hq, total_q, max_q_len, max_kv_len,
            float(scale), out.data_ptr(), _ptr(lse), workspace.data_ptr(), workspace.numel(),
            _stream(dev, stream)))
    else:
        rows = _rope_table(cos_sin, dev)
        _lib.check("rollout_attn_append_write_rope", lib.rollout_attn_append_write_rope(
            q.data_ptr(), k_new.data_ptr(), v_new.data_ptr(), cu_q.data_ptr(),
            ctx_lens.data_ptr(), ctypes.byref(s), B, Hq, total_q, max_q_len, max_kv_len,
            float(scale), cos_sin.data_ptr(), rows, out.data_ptr(), _ptr(lse),
            workspace.data_ptr(), workspace.numel(), _stream(dev, stream)))
    return out, lse


def append_workspace_size(B: int, Hq: int, Hkv: int, max_q_len: int) -> int:
    return int(_lib.load().rollout_attn_append_workspace_size(B, Hq, Hkv, max_q_len))


def mixed_workspace_size(B_decode: int, B_append: int, Hq: int, Hkv_decode: int,
                         Hkv_append: int, max_kv_len_decode: int, max_q_len: int) -> int:
    return int(_lib.load().rollout_attn_mixed_workspace_size(
        B_decode, B_append, Hq, Hkv_decode, Hkv_append, max_kv_len_decode, max_q_len))


def mixed(q_decode: torch.Tensor, kv_decode: PagedKV, kv_lens: torch.Tensor,
          q_append: torch.Tensor, cu_q: torch.Tensor, ctx_lens: torch.Tensor,
          kv_append: PagedKV, max_kv_len_decode: Optional[int] = None,
          max_q_len: Optional[int] = None, max_kv_len_append: Optional[int] = None,
          scale: Optional[float] = None, out_decode: Optional[torch.Tensor] = None,
          out_append: Optional[torch.Tensor] = None, want_lse: bool = False,
          workspace: Optional[torch.Tensor] = None, stream=None):
    """Decode rows and append rows of one step in one launch.

    q_decode bf16 [Bd][Hq][128] -> out_decode fp32 [Bd][Hq][128];
    q_append bf16 [total_q][Hq][128] -> out_append fp32 [total_q][Hq][128].
    Returns (out_decode, out_append, lse_decode, lse_append); the lse entries
    are None unless want_lse.
    """
    lib = _lib.load()
    dev = q_decode.device
    _need(q_decode, "q_decode", torch.bfloat16, dev)
    _need(kv_lens, "kv_lens", torch.int32, dev)
    _need(q_append, "q_append", torch.bfloat16, dev)
    _need(cu_q, "cu_q", torch.int32, dev)
    _need(ctx_lens, "ctx_lens", torch.int32, dev)
    for kv in (kv_decode, kv_append):
        if kv.device != dev:
            raise ValueError(f"caches must be on {dev}, got {kv.device}")
    Bd, Hq, D = q_decode.shape
    total_q = q_append.shape[0]
    _shape(q_decode, (Bd, Hq, HEAD_DIM), "q_decode")
    _shape(q_append, (total_q, Hq, HEAD_DIM), "q_append")
    _shape(kv_lens, (Bd,), "kv_lens")
    Ba = ctx_lens.shape[0]
    _shape(cu_q, (Ba + 1,), "cu_q")
    _rows(kv_decode, Bd)
    _rows(kv_append, Ba)
    if max_kv_len_decode is None:
        max_kv_len_decode = int(kv_lens.max().item()) if Bd else 0
    if max_q_len is None or max_kv_len_append is None:
        t = (cu_q[1:] - cu_q[:-1]) if Ba else cu_q[:0]
        if max_q_len is None:
            max_q_len = int(t.max().item()) if Ba else 0
        if max_kv_len_append is None:
            max_kv_len_append = int((t + ctx_lens).max().item()) if Ba else 0
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if out_decode is None:
        out_decode = _empty((Bd, Hq, D), torch.float32, dev, stream)
    if out_append is None:
        out_append = _empty((total_q, Hq, D), torch.float32, dev, stream)
    _need(out_decode, "out_decode", torch.float32, dev)
    _shape(out_decode, (Bd, Hq, HEAD_DIM), "out_decode")
    _need(out_append, "out_append", torch.float32, dev)
    _shape(out_append, (total_q, Hq, HEAD_DIM), "out_append")
    lse_d = _empty((Bd, Hq), torch.float32, dev, stream) if want_lse else None
    lse_a = _empty((total_q, Hq), torch.float32, dev, stream) if want_lse else None
    ws_bytes = lib.rollout_attn_mixed_workspace_size(
        Bd, Ba, Hq, kv_decode.num_kv_heads, kv_append.num_kv_heads, max_kv_len_decode,
        max_q_len)
    if workspace is None:
        workspace = _empty(max(ws_bytes, 1), torch.uint8, dev, stream)
    _need(workspace, "workspace", torch.uint8, dev)
    sd, sa = kv_decode.struct(), kv_append.struct()
    _lib.check("rollout_attn_mixed", lib.rollout_attn_mixed(
        q_decode.data_ptr(), ctypes.byref(sd), kv_lens.data_ptr(), Bd, max_kv_len_decode,
        out_decode.data_ptr(), _ptr(lse_d), q_append.data_ptr(), cu_q.data_ptr(),
        ctx_lens.data_ptr(), ctypes.byref(sa), Ba, total_q, max_q_len, max_kv_len_append,
        out_append.data_ptr(), _ptr(lse_a), Hq, float(scale), workspace.data_ptr(),
        workspace.numel(), _stream(dev, stream)))
    return out_decode, out_append, lse_d, lse_a


def _rope_table(cos_sin: torch.Tensor, dev) -> int:
    """Checks a rotary table (fp32 [rows][128]: cos | sin) and returns its rows."""
    _need(cos_sin, "cos_sin", torch.float32, dev)
    if cos_sin.dim() != 2 or cos_sin.shape[1] != HEAD_DIM:
        raise ValueError(f"cos_sin must have shape [rows][{HEAD_DIM}], got {tuple(cos_sin.shape)}")
    return int(cos_sin.shape[0])


def kv_page_write(k_new: torch.Tensor, v_new: torch.Tensor, cu_new: torch.Tensor,
                  start_pos: torch.Tensor, kv: PagedKV, max_new: Optional[int] = None,
                  max_pos: Optional[int] = None, stream=None,
                  cos_sin: Optional[torch.Tensor] = None) -> None:
    """Scatter packed new tokens (bf16 [N][Hkv][128]) into the pages (a bit copy into
    bf16 pools, quantized to E4M3 codes in fp8 pools). With a rotary table cos_sin
    (fp32 [rows][128], cos | sin per position) the keys are rotated at their
    positions as they are written."""
    lib = _lib.load()
    dev = kv.device
    _need(k_new, "k_new", torch.bfloat16, dev)
    _need(v_new, "v_new", torch.bfloat16, dev)
    _need(cu_new, "cu_new", torch.int32, dev)
    _need(start_pos, "start_pos", torch.int32, dev)
    B = start_pos.shape[0]
    _shape(cu_new, (B + 1,), "cu_new")
    _shape(k_new, (k_new.shape[0], kv.num_kv_heads, HEAD_DIM), "k_new")
    _shape(v_new, tuple(k_new.shape), "v_new")
    _rows(kv, B)
    if max_new is None or max_pos is None:
        n = (cu_new[1:] - cu_new[:-1]) if B else cu_new[:0]
        if max_new is None:
            max_new = int(n.max().item()) if B else 0
        if max_pos is None:
            max_pos = int((n + start_pos).max().item()) if B else 0
    s = kv.struct()
    if cos_sin is None:
        _lib.check("kv_page_write", lib.kv_page_write(
            k_new.data_ptr(), v_new.data_ptr(), cu_new.data_ptr(), start_pos.data_ptr(),
            ctypes.byref(s), B, k_new.shape[0], max_new, max_pos, _stream(dev, stream)))
    else:
        rows = _rope_table(cos_sin, dev)
        _lib.check("kv_page_write_rope", lib.kv_page_write_rope(
            k_new.data_ptr(), v_new.data_ptr(), cu_new.data_ptr(), start_pos.data_ptr(),
            ctypes.byref(s), B, k_new.shape[0], max_new, max_pos, cos_sin.data_ptr(), rows,
            _stream(dev, stream)))


def kv_page_gather(kv: PagedKV, lens: torch.Tensor, cu_out: torch.Tensor,
                   total: Optional[int] = None, max_len: Optional[int] = None, stream=None
                   ) -> Tuple[torch.Tensor, torch.Tensor]:
    """Copy logical tokens [0, lens[b]) of every row out to packed [total][Hkv][128]
    (bf16, or uint8 E4M3 codes for fp8 pools)."""
    lib = _lib.load()
    dev = kv.device
    _need(lens, "lens", torch.int32, dev)
    _need(cu_out, "cu_out", torch.int32, dev)
    B = lens.shape[0]
    _shape(cu_out, (B + 1,), "cu_out")
    _rows(kv, B)
    if total is None:
        total = int(cu_out[-1].item()) if B else 0
    if max_len is None:
        max_len = int(lens.max().item()) if B else 0
    k_out = _empty((total, kv.num_kv_heads, HEAD_DIM),
                   torch.uint8 if kv.fp8 else torch.bfloat16, dev, stream)
    v_out = _empty(tuple(k_out.shape), k_out.dtype, dev, stream)
    s = kv.struct()
    _lib.check("kv_page_gather", lib.kv_page_gather(
        ctypes.byref(s), lens.data_ptr(), cu_out.data_ptr(), B, total, max_len,
        k_out.data_ptr(), v_out.data_ptr(), _stream(dev, stream)))
    return k_out, v_out


def token_logprob_workspace_size(N: int, V: int, D: int) -> int:
    return int(_lib.load().token_logprob_workspace_size(N, V, D))


def _token_logprob(h, W, targets, scale, out, lse, want_lse, workspace, stream, packed_V):
    """Shared marshalling of token_logprob / token_logprob_packed (packed_V: V of a
    packed matrix, None for a row-major one)."""
    lib = _lib.load()
    dev = h.device
    _need(h, "h", torch.bfloat16, dev)
    _need(W, "W", torch.bfloat16, dev)
    _need(targets, "targets", torch.int32, dev)
    N, D = h.shape
    if packed_V is None:
        V = W.shape[0]
        _shape(W, (V, D), "W")
    else:
        V = int(packed_V)
        need = lib.token_logprob_packed_weight_size(V, D)
        if W.dim() != 1 or W.numel() * 2 < need:
            raise ValueError(f"W_packed: expected a flat bf16 tensor of {need // 2} elements "
                             f"for V={V}, D={D}, got {tuple(W.shape)}")
    _shape(targets, (N,), "targets")
    if out is None:
        out = _empty((N,), torch.float32, dev, stream)
    _need(out, "out", torch.float32, dev)
    _shape(out, (N,), "out")
    if lse is None and want_lse:
        lse = _empty((N,), torch.float32, dev, stream)
    if lse is not None:
        _need(lse, "lse", torch.float32, dev)
        _shape(lse, (N,), "lse")
    if workspace is None:
        workspace = _empty(max(lib.token_logprob_workspace_size(N, V, D), 1), torch.uint8, dev,
                           stream)
    _need(workspace, "workspace", torch.uint8, dev)
    fn = lib.token_logprob if packed_V is None else lib.token_logprob_packed
    name = "token_logprob" if packed_V is None else "token_logprob_packed"
    _lib.check(name, fn(
        h.data_ptr(), W.data_ptr(), targets.data_ptr(), N, V, D, float(scale), out.data_ptr(),
        _ptr(lse), workspace.data_ptr(), workspace.numel(), _stream(dev, stream)))
    return out, lse


def token_logprob(h: torch.Tensor, W: torch.Tensor, targets: torch.Tensor, scale: float = 1.0,
                  out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                  want_lse: bool = False, workspace: Optional[torch.Tensor] = None, stream=None
                  ) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """Log-probability of targets[n] under logits scale * h[n] . W^T.

    h bf16 [N][D], W bf16 [V][D], targets int32 [N] -> logprob fp32 [N] (, lse fp32 [N]).
    """
    return _token_logprob(h, W, targets, scale, out, lse, want_lse, workspace, stream, None)


def token_logprob_pack_weight(W: torch.Tensor, out: Optional[torch.Tensor] = None,
                              stream=None) -> torch.Tensor:
    """Packed copy of the LM-head matrix W bf16 [V][D] for token_logprob_packed
    (a flat bf16 tensor; rows past V are zeros)."""
    lib = _lib.load()
    dev = W.device
    _need(W, "W", torch.bfloat16, dev)
    V, D = W.shape
    n = lib.token_logprob_packed_weight_size(V, D) // 2
    if out is None:
        out = _empty((max(n, 1),), torch.bfloat16, dev, stream)
    _need(out, "out", torch.bfloat16, dev)
    _lib.check("token_logprob_pack_weight", lib.token_logprob_pack_weight(
        W.data_ptr(), V, D, out.data_ptr(), out.numel() * 2, _stream(dev, stream)))
    return out


def token_logprob_packed(h: torch.Tensor, W_packed: torch.Tensor, V: int, targets: torch.Tensor,
                         scale: float = 1.0, out: Optional[torch.Tensor] = None,
                         lse: Optional[torch.Tensor] = None, want_lse: bool = False,
                         workspace: Optional[torch.Tensor] = None, stream=None
                         ) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """token_logprob with the packed matrix from token_logprob_pack_weight (V rows)."""
    return _token_logprob(h, W_packed, targets, scale, out, lse, want_lse, workspace, stream, V)
