"""ctypes binding of the hardware-ceiling microbenchmarks (include/ra_microbench.h).

Each function launches on torch's current stream, waits for it and returns the
measured figure; the benchmark reports them beside the vendor peaks.
"""
import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libra_microbench.so")
EXPORTS = ("ra_mb_mfma_bf16", "ra_mb_lds_read", "ra_mb_stream_read", "ra_mb_block_read",
           "ra_mb_l2_read")
MFMA_THREADS = 256
MFMA_OPERANDS = MFMA_THREADS * 64
LDS_THREADS = 512
_lib = None


def load() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2603_18815_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        i32, i64, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
        lib.ra_mb_mfma_bf16.argtypes = [vp, i32, i32, vp, vp, vp]
        lib.ra_mb_lds_read.argtypes = [i32, i32, vp, vp, vp]
        lib.ra_mb_stream_read.argtypes = [vp, i64, vp, i32, vp, vp]
        lib.ra_mb_block_read.argtypes = [vp, i64, i32, i32, vp, vp]
        lib.ra_mb_l2_read.argtypes = [vp, i64, i32, i32, i32, vp, vp]
        for f in EXPORTS:
            getattr(lib, f).restype = ctypes.c_int
        _lib = lib
    return _lib


def _check(name, rc):
    if rc != 0:
        raise RuntimeError(f"{name} returned {rc}")


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _clock_ghz(clocks: torch.Tensor) -> float:
    c = clocks.cpu().tolist()
    return (c[2] - c[0]) / max(c[3] - c[1], 1) * 0.1   # real-time counter ticks at 100 MHz


def mfma_bf16(blocks: int, iters: int, zeros: bool = False, seed: int = 0, reps: int = 3):
    """Rate of v_mfma_f32_32x32x16_bf16 with 4 independent accumulators per wave.

    Returns (TFLOP/s from HIP events, shader clock in GHz while the products ran)."""
    lib = load()
    dev = torch.device("cuda", torch.cuda.current_device())
    g = torch.Generator(device=dev).manual_seed(seed)
    ops = (torch.zeros(MFMA_OPERANDS, device=dev, dtype=torch.bfloat16) if zeros else
           (torch.rand(MFMA_OPERANDS, device=dev, generator=g) * 2 - 1).to(torch.bfloat16))
    sink = torch.empty(blocks * MFMA_THREADS, device=dev, dtype=torch.float32)
    clocks = torch.zeros(4, device=dev, dtype=torch.int64)
    run = lambda: _check("ra_mb_mfma_bf16", lib.ra_mb_mfma_bf16(
        ops.data_ptr(), blocks, iters, sink.data_ptr(), clocks.data_ptr(), _stream()))
    run()
    best = None
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        run()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None else min(best, ms)
    flops = blocks * 4 * iters * 4 * 32768
    return flops / (best * 1e-3) / 1e12, _clock_ghz(clocks)


def lds_read(blocks: int, iters: int, reps: int = 3):
    """LDS read bandwidth. Returns (bytes per shader clock per workgroup of the first
    compute unit's timer wave, shader clock in GHz, aggregate GB/s from HIP events)."""
    lib = load()
    dev = torch.device("cuda", torch.cuda.current_device())
    sink = torch.empty(blocks * LDS_THREADS, device=dev, dtype=torch.int32)
    clocks = torch.zeros(4, device=dev, dtype=torch.int64)
    run = lambda: _check("ra_mb_lds_read", lib.ra_mb_lds_read(
        blocks, iters, sink.data_ptr(), clocks.data_ptr(), _stream()))
    run()
    best = None
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        run()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None else min(best, ms)
    c = clocks.cpu().tolist()
    per_block = LDS_THREADS * iters * 128
    return per_block / max(c[2] - c[0], 1), _clock_ghz(clocks), \
        blocks * per_block / (best * 1e-3) / 1e9


def stream_read(nbytes: int, paged: bool, blocks: int, seed: int = 0, reps: int = 5):
    """HBM read rate (GB/s) of one pass over nbytes, in address order or in a
    shuffled order of 4 KiB blocks."""
    lib = load()
    dev = torch.device("cuda", torch.cuda.current_device())
    src = torch.empty(nbytes, device=dev, dtype=torch.uint8)
    src.fill_(1)
    order = None
    if paged:
        g = torch.Generator(device=dev).manual_seed(seed)
        order = torch.randperm(nbytes // 4096, device=dev, generator=g).to(torch.int32)
    sink = torch.empty(blocks * 256, device=dev, dtype=torch.int32)
    run = lambda: _check("ra_mb_stream_read", lib.ra_mb_stream_read(
        src.data_ptr(), nbytes, None if order is None else order.data_ptr(), blocks,
        sink.data_ptr(), _stream()))
    run()
    ms = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        run()
        e1.record()
        torch.cuda.synchronize()
        ms.append(e0.elapsed_time(e1))
    best = min(ms)
    extra = 0 if order is None else order.numel() * 4
    return (nbytes + extra) / (best * 1e-3) / 1e9


def block_read(src: torch.Tensor, block_bytes: int, blocks: int, reps: int = 5):
    """HBM read rate (GB/s) of one pass over src (uint8, device; its size a power-of-two
    multiple of block_bytes) in shuffled blocks of block_bytes (1, 2 or 4 KiB)."""
    lib = load()
    sink = torch.empty(blocks * 256, device=src.device, dtype=torch.int32)
    run = lambda: _check("ra_mb_block_read", lib.ra_mb_block_read(
        src.data_ptr(), src.numel(), block_bytes, blocks, sink.data_ptr(), _stream()))
    run()
    ms = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        run()
        e1.record()
        torch.cuda.synchronize()
        ms.append(e0.elapsed_time(e1))
    return src.numel() / (min(ms) * 1e-3) / 1e9


def l2_read(to_lds: bool, blocks: int, iters: int, nbytes: int = 1 << 21, reps: int = 3):
    """Rate (GB/s, best of reps) at which the L2 feeds the compute units: an
    nbytes buffer (it stays in each XCD's L2) read over and over, by direct
    global-to-LDS loads (to_lds) or loads into registers."""
    lib = load()
    dev = torch.device("cuda", torch.cuda.current_device())
    src = torch.zeros(nbytes, device=dev, dtype=torch.uint8)
    sink = torch.empty(blocks * 256, device=dev, dtype=torch.int32)
    run = lambda: _check("ra_mb_l2_read", lib.ra_mb_l2_read(
        src.data_ptr(), nbytes, int(to_lds), blocks, iters, sink.data_ptr(), _stream()))
    run()
    best = None
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        run()
        e1.record()
        torch.cuda.synchronize()
        gbs = blocks * iters * 65536 / (e0.elapsed_time(e1) * 1e6)
        best = gbs if best is None else max(best, gbs)
    return best
