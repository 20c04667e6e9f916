"""fp64 CPU oracle for paged rollout attention (TEST INFRASTRUCTURE).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package. It shares no code with the HIP library
(`paper_2603_18815_amd`) and never imports it.

The arithmetic lives in `attn_oracle.c` and `logprob_oracle.c` (plain loops,
fp64, libm exp/log); this module only marshals numpy arrays into it. What each function computes and the
readings it adopts where the paper is silent are stated at the top of that file.
Every function here is pinned by the `-m "not gpu"` tests in
`tests/test_oracle_pins.py` (library routine, closed forms, invariants, brute
force, hand-derived fixtures under `tests/golden/`).
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None

_u16p = np.ctypeslib.ndpointer(dtype=np.uint16, flags="C_CONTIGUOUS")
_i32p = np.ctypeslib.ndpointer(dtype=np.int32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(dtype=np.float64, flags="C_CONTIGUOUS")
_u8p = np.ctypeslib.ndpointer(dtype=np.uint8, flags="C_CONTIGUOUS")


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_build.LIB) or any(
        os.path.getmtime(_build.LIB) < os.path.getmtime(src) for src in _build.SRCS
    ):
        _build.build()
    lib = ctypes.CDLL(_build.LIB)
    c_i64, c_int, c_dbl = ctypes.c_int64, ctypes.c_int, ctypes.c_double
    lib.oracle_decode_f64.argtypes = [_u16p, _u16p, _u16p, _i32p, c_i64, _i32p, c_int, c_int,
                                      c_int, c_int, c_int, c_dbl, _f64p, _f64p]
    lib.oracle_decode_f64.restype = c_int
    lib.oracle_set_num_threads.argtypes = [c_int]
    lib.oracle_set_num_threads.restype = None
    lib.oracle_append_f64.argtypes = [_u16p, _i32p, _i32p, _u16p, _u16p, _i32p, c_i64, c_int,
                                      c_int, c_int, c_int, c_int, c_dbl, _f64p, _f64p]
    lib.oracle_append_f64.restype = c_int
    lib.oracle_page_write.argtypes = [_u16p, _u16p, _i32p, _i32p, _i32p, c_i64, c_int, c_int,
                                      c_int, c_int, _u16p, _u16p]
    lib.oracle_page_write.restype = c_int
    lib.oracle_page_gather.argtypes = [_u16p, _u16p, _i32p, c_i64, _i32p, _i32p, c_int, c_int,
                                       c_int, c_int, _u16p, _u16p]
    lib.oracle_page_gather.restype = c_int
    lib.oracle_token_logprob_f64.argtypes = [_u16p, _u16p, _i32p, c_i64, c_i64, c_i64, c_dbl,
                                             _f64p, _f64p]
    lib.oracle_token_logprob_f64.restype = c_int
    c_flt = ctypes.c_float
    lib.oracle_decode_fp8_f64.argtypes = [_u16p, _u8p, _u8p, c_dbl, c_dbl, _i32p, c_i64, _i32p,
                                          c_int, c_int, c_int, c_int, c_int, c_dbl, _f64p, _f64p]
    lib.oracle_decode_fp8_f64.restype = c_int
    lib.oracle_append_fp8_f64.argtypes = [_u16p, _i32p, _i32p, _u8p, _u8p, c_dbl, c_dbl, _i32p,
                                          c_i64, c_int, c_int, c_int, c_int, c_int, c_dbl, _f64p,
                                          _f64p]
    lib.oracle_append_fp8_f64.restype = c_int
    lib.oracle_page_write_fp8.argtypes = [_u16p, _u16p, _i32p, _i32p, _i32p, c_i64, c_int, c_int,
                                          c_int, c_int, c_flt, c_flt, _u8p, _u8p]
    lib.oracle_page_write_fp8.restype = c_int
    lib.oracle_page_gather_u8.argtypes = [_u8p, _u8p, _i32p, c_i64, _i32p, _i32p, c_int, c_int,
                                          c_int, c_int, _u8p, _u8p]
    lib.oracle_page_gather_u8.restype = c_int
    lib.oracle_e4m3_decode.argtypes = [_u8p, c_i64, _f64p]
    lib.oracle_e4m3_decode.restype = None
    lib.oracle_e4m3_encode.argtypes = [_f64p, c_i64, _u8p]
    lib.oracle_e4m3_encode.restype = None
    lib.oracle_rope_bf16.argtypes = [_u16p, c_i64, c_int, _i32p,
                                     np.ctypeslib.ndpointer(dtype=np.float32,
                                                            flags="C_CONTIGUOUS"),
                                     c_i64, _u16p]
    lib.oracle_rope_bf16.restype = c_int
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = c_int
    _lib = lib
    return lib


def num_threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Set the OpenMP threads of the oracle's parallel loops (timing only)."""
    _load().oracle_set_num_threads(int(n))


def _u16(a):
    a = np.asarray(a)
    if a.dtype != np.uint16:
        raise TypeError("bf16 data must be passed as uint16 bit patterns")
    return np.ascontiguousarray(a)


def _i32(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def pool_dims(k_pool, v_pool, page_size, head_dim):
    """(num_pages, Hkv) of a pool pair; K is [pages][Hkv][P][D], V is [pages][Hkv][D][P]."""
    if k_pool.ndim != 4 or v_pool.ndim != 4:
        raise ValueError("pools must be 4-D")
    n, hkv, p, d = k_pool.shape
    if (p, d) != (page_size, head_dim) or v_pool.shape != (n, hkv, head_dim, page_size):
        raise ValueError(f"pool shapes {k_pool.shape} / {v_pool.shape} do not match the layout")
    return n, hkv


def decode(q, k_pool, v_pool, block_table, kv_lens, scale):
    """Decode attention, fp64. q bf16 bits [B][Hq][D]; returns (out [B][Hq][D], lse [B][Hq])."""
    lib = _load()
    q = _u16(q)
    k_pool, v_pool = _u16(k_pool), _u16(v_pool)
    B, Hq, D = q.shape
    P = k_pool.shape[2]
    _, Hkv = pool_dims(k_pool, v_pool, P, D)
    bt = _i32(block_table)
    lens = _i32(kv_lens)
    out = np.zeros((B, Hq, D), np.float64)
    lse = np.zeros((B, Hq), np.float64)
    rc = lib.oracle_decode_f64(q, k_pool, v_pool, bt, bt.shape[1] if bt.ndim == 2 else 0, lens,
                               B, Hq, Hkv, P, D, float(scale), out, lse)
    if rc != 0:
        raise RuntimeError(f"oracle_decode_f64 failed ({rc})")
    return out, lse


def append(q, cu_q, ctx_lens, k_pool, v_pool, block_table, scale):
    """Append attention, fp64. q bf16 bits [total_q][Hq][D]; returns (out, lse)."""
    lib = _load()
    q = _u16(q)
    k_pool, v_pool = _u16(k_pool), _u16(v_pool)
    total_q, Hq, D = q.shape
    P = k_pool.shape[2]
    _, Hkv = pool_dims(k_pool, v_pool, P, D)
    cu = _i32(cu_q)
    ctx = _i32(ctx_lens)
    B = ctx.shape[0]
    if cu.shape[0] != B + 1 or cu[-1] != total_q:
        raise ValueError("cu_q must have B+1 entries ending at total_q")
    bt = _i32(block_table)
    out = np.zeros((total_q, Hq, D), np.float64)
    lse = np.zeros((total_q, Hq), np.float64)
    rc = lib.oracle_append_f64(q, cu, ctx, k_pool, v_pool, bt, bt.shape[1] if bt.ndim == 2 else 0,
                               B, Hq, Hkv, P, D, float(scale), out, lse)
    if rc != 0:
        raise RuntimeError(f"oracle_append_f64 failed ({rc})")
    return out, lse


def page_write(k_new, v_new, cu_new, start_pos, block_table, k_pool, v_pool):
    """Return copies of (k_pool, v_pool) with the new tokens scattered in (bit copy)."""
    lib = _load()
    k_new, v_new = _u16(k_new), _u16(v_new)
    kp, vp = _u16(k_pool).copy(), _u16(v_pool).copy()
    P, D = kp.shape[2], kp.shape[3]
    _, Hkv = pool_dims(kp, vp, P, D)
    cu = _i32(cu_new)
    sp = _i32(start_pos)
    bt = _i32(block_table)
    rc = lib.oracle_page_write(k_new, v_new, cu, sp, bt, bt.shape[1], sp.shape[0], Hkv, P, D,
                               kp, vp)
    if rc != 0:
        raise RuntimeError(f"oracle_page_write failed ({rc})")
    return kp, vp


def page_gather(k_pool, v_pool, block_table, lens, cu_out):
    """Logical tokens [0, lens[b]) of every row, packed token-major: (k [total][Hkv][D], v)."""
    lib = _load()
    kp, vp = _u16(k_pool), _u16(v_pool)
    P, D = kp.shape[2], kp.shape[3]
    _, Hkv = pool_dims(kp, vp, P, D)
    lens = _i32(lens)
    cu = _i32(cu_out)
    bt = _i32(block_table)
    total = int(cu[-1]) if cu.size else 0
    k_out = np.zeros((total, Hkv, D), np.uint16)
    v_out = np.zeros((total, Hkv, D), np.uint16)
    rc = lib.oracle_page_gather(kp, vp, bt, bt.shape[1], lens, cu, lens.shape[0], Hkv, P, D,
                                k_out, v_out)
    if rc != 0:
        raise RuntimeError(f"oracle_page_gather failed ({rc})")
    return k_out, v_out


def token_logprob(h, W, targets, scale=1.0):
    """Per-token log-probability of targets[n] under logits scale * h[n] . W^T.

    h: uint16 bf16 bits [N][D]; W: uint16 bf16 bits [V][D]; targets: int [N].
    Returns (logp [N], lse [N]) in fp64; logp is NaN for a target outside [0, V).
    """
    h = np.ascontiguousarray(h, np.uint16)
    W = np.ascontiguousarray(W, np.uint16)
    t = np.ascontiguousarray(targets, np.int32)
    N, D = h.shape
    V = W.shape[0]
    assert W.shape[1] == D and t.shape == (N,)
    logp = np.empty(N, np.float64)
    lse = np.empty(N, np.float64)
    rc = _load().oracle_token_logprob_f64(h, W, t, N, V, D, float(scale), logp, lse)
    assert rc == 0
    return logp, lse


# --------------------------------------------------------------------------- fp8 pools

def _u8(a):
    a = np.asarray(a)
    if a.dtype != np.uint8:
        raise TypeError("fp8 pools must be passed as uint8 E4M3 codes")
    return np.ascontiguousarray(a)


def e4m3_decode(codes):
    """OCP E4M3 codes (uint8) -> values (fp64; NaN for 0x7F / 0xFF)."""
    c = _u8(codes)
    out = np.empty(c.shape, np.float64)
    _load().oracle_e4m3_decode(c.reshape(-1), c.size, out.reshape(-1))
    return out


def e4m3_encode(x):
    """Values -> OCP E4M3 codes: nearest finite code, ties to the even code, +-inf and
    magnitudes beyond 448 saturated to +-448, NaN to 0x7F."""
    v = np.ascontiguousarray(np.asarray(x, np.float64))
    out = np.empty(v.shape, np.uint8)
    _load().oracle_e4m3_encode(v.reshape(-1), v.size, out.reshape(-1))
    return out


def quantize(x_bits, scale):
    """The code a pool with this scale stores for bf16 values x: encode(fp32(x) * fp32(1/scale))."""
    x = _u16(x_bits)
    f = (x.astype(np.uint32) << 16).view(np.float32)
    inv = np.float32(1.0) / np.float32(scale)
    # inf / NaN inputs and fp32 overflow are meant (IEEE results; the encoder
    # saturates infinities and maps NaN to its NaN code)
    with np.errstate(over="ignore", invalid="ignore"):
        y = (f * inv).astype(np.float32)
    return e4m3_encode(y)


def page_write_fp8(k_new, v_new, cu_new, start_pos, block_table, k_pool, v_pool, k_scale,
                   v_scale):
    """Return copies of fp8 pools (k_pool, v_pool) with the new bf16 tokens quantized in."""
    lib = _load()
    k_new, v_new = _u16(k_new), _u16(v_new)
    kp, vp = _u8(k_pool).copy(), _u8(v_pool).copy()
    P, D = kp.shape[2], kp.shape[3]
    _, Hkv = pool_dims(kp, vp, P, D)
    cu, sp, bt = _i32(cu_new), _i32(start_pos), _i32(block_table)
    rc = lib.oracle_page_write_fp8(k_new, v_new, cu, sp, bt, bt.shape[1], sp.shape[0], Hkv, P, D,
                                   float(k_scale), float(v_scale), kp, vp)
    if rc != 0:
        raise RuntimeError(f"oracle_page_write_fp8 failed ({rc})")
    return kp, vp


def page_gather_u8(k_pool, v_pool, block_table, lens, cu_out):
    """Stored codes of logical tokens [0, lens[b]) of every row, packed token-major."""
    lib = _load()
    kp, vp = _u8(k_pool), _u8(v_pool)
    P, D = kp.shape[2], kp.shape[3]
    _, Hkv = pool_dims(kp, vp, P, D)
    lens, cu, bt = _i32(lens), _i32(cu_out), _i32(block_table)
    total = int(cu[-1]) if cu.size else 0
    k_out = np.zeros((total, Hkv, D), np.uint8)
    v_out = np.zeros((total, Hkv, D), np.uint8)
    rc = lib.oracle_page_gather_u8(kp, vp, bt, bt.shape[1], lens, cu, lens.shape[0], Hkv, P, D,
                                   k_out, v_out)
    if rc != 0:
        raise RuntimeError(f"oracle_page_gather_u8 failed ({rc})")
    return k_out, v_out


def decode_fp8(q, k_pool, v_pool, k_scale, v_scale, block_table, kv_lens, scale):
    """Decode attention over fp8 pools (values code * k_scale, code * v_scale), fp64."""
    lib = _load()
    q = _u16(q)
    kp, vp = _u8(k_pool), _u8(v_pool)
    B, Hq, D = q.shape
    P = kp.shape[2]
    _, Hkv = pool_dims(kp, vp, P, D)
    bt, lens = _i32(block_table), _i32(kv_lens)
    out = np.zeros((B, Hq, D), np.float64)
    lse = np.zeros((B, Hq), np.float64)
    rc = lib.oracle_decode_fp8_f64(q, kp, vp, float(k_scale), float(v_scale), bt,
                                   bt.shape[1] if bt.ndim == 2 else 0, lens, B, Hq, Hkv, P, D,
                                   float(scale), out, lse)
    if rc != 0:
        raise RuntimeError(f"oracle_decode_fp8_f64 failed ({rc})")
    return out, lse


def append_fp8(q, cu_q, ctx_lens, k_pool, v_pool, k_scale, v_scale, block_table, scale):
    """Append attention over fp8 pools, fp64. Returns (out, lse)."""
    lib = _load()
    q = _u16(q)
    kp, vp = _u8(k_pool), _u8(v_pool)
    total_q, Hq, D = q.shape
    P = kp.shape[2]
    _, Hkv = pool_dims(kp, vp, P, D)
    cu, ctx, bt = _i32(cu_q), _i32(ctx_lens), _i32(block_table)
    B = ctx.shape[0]
    if cu.shape[0] != B + 1 or cu[-1] != total_q:
        raise ValueError("cu_q must have B+1 entries ending at total_q")
    out = np.zeros((total_q, Hq, D), np.float64)
    lse = np.zeros((total_q, Hq), np.float64)
    rc = lib.oracle_append_fp8_f64(q, cu, ctx, kp, vp, float(k_scale), float(v_scale), bt,
                                   bt.shape[1] if bt.ndim == 2 else 0, B, Hq, Hkv, P, D,
                                   float(scale), out, lse)
    if rc != 0:
        raise RuntimeError(f"oracle_append_fp8_f64 failed ({rc})")
    return out, lse


def rope(x, positions, cos_sin):
    """Rows x (bf16 bits [N][H][128]) rotated at positions [N] with the rotary table
    cos_sin (fp32 [rows][128]: cos | sin), as bf16 bits (see attn_oracle.c)."""
    lib = _load()
    x = _u16(x)
    N, H, D = x.shape
    assert D == 128
    pos = _i32(positions).reshape(-1)
    assert pos.shape[0] == N
    cs = np.ascontiguousarray(np.asarray(cos_sin, np.float32))
    out = np.empty_like(x)
    if lib.oracle_rope_bf16(x, N, H, pos, cs, cs.shape[0], out) != 0:
        raise ValueError("rope: a position lies outside the table")
    return out
