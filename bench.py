#!/usr/bin/env python3
"""Benchmark of one rollout-attention step on one MI355X.

A step is one pass of the whole hot path over one batch of seeded synthetic
input at the Qwen3-8B GQA shape (Hq = 32, Hkv = 8, head dim 128, 16-token
pages, bf16 K/V, fp32 outputs):
  1. kv_page_write  - the step's new tokens: one decode token per decode row
                      and every append row's observation chunk;
  2. rollout_attn_append - B = 32 trajectories, cached context uniform in
                      [2048, 24576], chunk uniform in [64, 2048] tokens;
  3. rollout_attn_decode - B = 64 trajectories, context uniform in
                      [4096, 32768] keys, shuffled pages (split + combine kernels).
Append runs before decode (the two are independent): the page write leaves
its new tokens as dirty cache lines, and their write-back then overlaps the
matrix-bound append instead of the HBM-bound decode.
Inputs are resident in HBM before timing starts. Each call is bracketed by HIP
events on the stream the library launches on (torch's current stream).

Printed: one JSON line. `value` is the decode attention's algorithmic HBM
GB/s (K/V bytes of every attended key + q + out + block table + lengths,
divided by the decode call's time); the append's algorithmic TFLOP/s (only
unmasked query-key pairs, two matrix products each) is reported beside it.
`roofline` is the decode kernel pair against the 8 TB/s HBM peak,
`roofline_append` the append kernel against the 2.5 PFLOP/s dense bf16 peak.
`mixed_step` times the mixed rollout step on one pool (B = 512 trajectories,
85 % decode rows / 15 % append rows, log-normal contexts: page write, append,
decode on one stream) beside its lower bounds at the published peaks, and the
same step with decode and append rows in one persistent launch
(`single_launch`).
`append_write` times the append workload's page write + append as two calls
and as one fused call.
`fp8_kv_decode` times the decode workload (and the append workload) over fp8
(OCP E4M3) pools beside the bf16 pools (each alone).
`shared_prefix_decode` times plain and shared-prefix decode of 8 tasks x 8
rollouts whose rows share each task's prompt pages. `token_logprob` times the
fused LM-head log-probability kernel at the Qwen3-8B head for 64 and 1024
tokens, with the head row-major and packed.
`long_horizon_decode` times decode of B = 256 trajectories with Hq = 64 and
contexts log-normal around 16384 keys (up to 65536). `achievable` gives what this
GPU delivers to the kernels, measured in the same run (matrix-core rate and
clock, LDS reads, streaming and paged HBM reads).
`cpu_baseline` is the fp64 CPU oracle on a bounded sample of the same inputs
(`cpu_baseline_single_thread`: the small decode workload on one thread;
`cpu_baseline_long_decode`: whole rows of the long-horizon workload).
"""
import argparse
import json
import math
import os
import sys
import time

import numpy as np

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
SCALE = 1.0 / math.sqrt(128)


def decode_bytes(w) -> int:
    L = w.kv_lens.astype(np.int64)
    D = w.head_dim
    per_row = (L * w.Hkv * D * 2 * 2 + w.Hq * D * 2 + w.Hq * D * 4
               + 4 * ((L + w.page_size - 1) // w.page_size) + 4)
    return int(per_row.sum())


def append_flops(w) -> int:
    T = w.q_lens.astype(np.int64)
    C = w.ctx_lens.astype(np.int64)
    return int(4 * w.head_dim * w.Hq * (T * C + T * (T + 1) // 2).sum())


def write_bytes(n_new: int, Hkv: int, D: int = 128) -> int:
    return 2 * n_new * Hkv * D * 2 * 2


ROOT = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCES = {
    "decode": ("paper_2603_18815_amd/csrc/ra_decode.hip",
               "paper_2603_18815_amd/csrc/ra_decode_split.h",
               "paper_2603_18815_amd/csrc/ra_device.h"),
    "append": ("paper_2603_18815_amd/csrc/ra_persistent.hip",
               "paper_2603_18815_amd/csrc/ra_append_tile.h",
               "paper_2603_18815_amd/csrc/ra_device.h"),
}
KERNEL_SOURCES["long_decode"] = KERNEL_SOURCES["decode"]
TRAFFIC_FILES = {
    "decode": "profiles/decode_qwen3_8b_b64.hbm_traffic.txt",
    "append": "profiles/append_qwen3_8b_b32.hbm_traffic.txt",
    "long_decode": "profiles/decode_long_horizon_b256.hbm_traffic.txt",
}


def measured_traffic(part: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or None
    when there is none or the kernel source has changed since it was taken."""
    import hashlib
    path = os.path.join(ROOT, TRAFFIC_FILES[part])
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if "=" in line and not line.startswith("#"):
            k, v = line.split("#")[0].split("=", 1)
            fields[k.strip()] = v.strip()
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[part]:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    if fields.get("source_sha256_16") != h.hexdigest()[:16]:
        return None
    return int(float(fields["hbm_bytes_per_launch"]))


def cpu_baseline(wd, td, wa, ta, seconds: float):
    """Time the fp64 oracle on bounded samples of the benchmark's own inputs."""
    import oracle
    import torch
    from synth import bits, compact_rows

    cores = oracle.num_threads()
    cpu_model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    # decode: whole rows of the decode workload, taken in a fixed order until the budget
    rng = np.random.default_rng(0)
    order = rng.permutation(wd.kv_lens.shape[0])
    dev = td.k_pool.device
    done_bytes, spent, rows_done, passes = 0, 0.0, 0, 0
    table = wd.decode_table()
    # whole passes over the workload (in 8 chunks of rows) until the budget is spent
    chunks = [(chunk, compact_rows(td.k_pool, td.v_pool, table[chunk], wd.kv_lens[chunk]),
               bits(td.q_decode[torch.as_tensor(chunk, device=dev)]))
              for chunk in np.array_split(order, 8)]
    while spent <= seconds and passes < 64:
        for chunk, (k, v, bt), q in chunks:
            t0 = time.perf_counter()
            oracle.decode(q, k, v, bt, wd.kv_lens[chunk], SCALE)
            spent += time.perf_counter() - t0
            sub = wd.kv_lens[chunk].astype(np.int64)
            done_bytes += int((sub * wd.Hkv * 128 * 4 + wd.Hq * 128 * 6
                               + 4 * ((sub + 15) // 16) + 4).sum())
            rows_done += len(chunk)
            if spent > seconds:
                break
        passes += 1
    del chunks
    dec = {"value": done_bytes / spent / 1e9, "unit": "GB/s", "cores": cores, "kind": "oracle",
           "cpu_model": cpu_model,
           "sample": f"decode, {rows_done} rows ({rows_done / wd.kv_lens.shape[0]:.2f} passes "
                     f"over the {wd.kv_lens.shape[0]} rows of the decode workload, all heads), "
                     f"{spent:.1f} s wall"}
    # append: single queries (query i of a row == a one-token chunk at ctx + i),
    # drawn in batches of 64 from random rows until the time budget is spent
    cu = wa.cu_q()
    spent_a, flops, nq = 0.0, 0, 0
    while spent_a < seconds and nq < 4096:
        qs, ctx1, rows = [], [], []
        for r in rng.integers(0, wa.q_lens.shape[0], 64):
            i = int(rng.integers(0, int(wa.q_lens[r])))
            qs.append(int(cu[r]) + i)
            ctx1.append(int(wa.ctx_lens[r]) + i)
            rows.append(int(r))
        ctx1 = np.array(ctx1, np.int32)
        k, v, bt = compact_rows(ta.k_pool, ta.v_pool, wa.append_table()[np.array(rows)], ctx1 + 1)
        q = bits(ta.q_append[torch.as_tensor(qs, device=dev)])
        t0 = time.perf_counter()
        oracle.append(q, np.arange(len(qs) + 1, dtype=np.int32), ctx1, k, v, bt, SCALE)
        spent_a += time.perf_counter() - t0
        flops += 4 * 128 * wa.Hq * int((ctx1.astype(np.int64) + 1).sum())
        nq += len(qs)
    app = {"value": flops / spent_a / 1e12, "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
           "cpu_model": cpu_model,
           "sample": f"append, {nq} single queries (all heads) drawn from random rows of the "
                     f"append workload, {spent_a:.1f} s wall"}
    # the small decode workload (B = 4, Hq = 8, Hkv = 2) in full, on one thread
    import synth
    w1 = synth.config(1)
    t1 = synth.make_tensors(w1, dev)
    k1, v1, bt1 = compact_rows(t1.k_pool, t1.v_pool, w1.decode_table(), w1.kv_lens)
    q1 = bits(t1.q_decode)
    del t1
    oracle.set_num_threads(1)
    try:
        spent1, reps = 0.0, 0
        while spent1 < min(seconds, 2.0):
            t0 = time.perf_counter()
            oracle.decode(q1, k1, v1, bt1, w1.kv_lens, SCALE)
            spent1 += time.perf_counter() - t0
            reps += 1
    finally:
        oracle.set_num_threads(cores)
    single = {"value": decode_bytes(w1) * reps / spent1 / 1e9, "unit": "GB/s", "cores": 1,
              "kind": "oracle", "cpu_model": cpu_model,
              "sample": f"decode, the whole B=4 workload ({w1.name}) {reps} times on one thread, "
                        f"{spent1:.2f} s wall"}
    # the long-horizon decode workload (B = 256, Hq = 64): whole rows in a seeded order
    w4 = synth.config(4)
    t4 = synth.make_tensors(w4, dev)
    order4 = np.random.default_rng(4).permutation(w4.kv_lens.shape[0])
    table4 = w4.decode_table()
    spent4, bytes4, rows4 = 0.0, 0, 0
    for chunk in np.array_split(order4, 32):
        k4, v4, bt4 = compact_rows(t4.k_pool, t4.v_pool, table4[chunk], w4.kv_lens[chunk])
        q4 = bits(t4.q_decode[torch.as_tensor(chunk, device=dev)])
        t0 = time.perf_counter()
        oracle.decode(q4, k4, v4, bt4, w4.kv_lens[chunk], SCALE)
        spent4 += time.perf_counter() - t0
        sub = w4.kv_lens[chunk].astype(np.int64)
        bytes4 += int((sub * w4.Hkv * 128 * 4 + w4.Hq * 128 * 6 + 4 * ((sub + 15) // 16)
                       + 4).sum())
        rows4 += len(chunk)
        del k4, v4, q4
        if spent4 > seconds:
            break
    del t4
    torch.cuda.empty_cache()
    long4 = {"value": bytes4 / spent4 / 1e9, "unit": "GB/s", "cores": cores, "kind": "oracle",
             "cpu_model": cpu_model,
             "sample": f"decode, {rows4} whole rows (all 64 heads) of the {w4.kv_lens.shape[0]}-row "
                       f"long-horizon workload in a seeded order, {spent4:.1f} s wall"}
    return dec, app, single, long4


def long_decode_leg(ra, synth, dev, steps: int, warmup: int):
    """Decode of the long-horizon workload: B = 256 trajectories, Hq = 64, Hkv = 8,
    contexts log-normal around 16384 keys clipped to [512, 65536], shuffled pages
    (split + combine kernels, one call per step)."""
    import torch

    w = synth.config(4)
    t = synth.make_tensors(w, dev)
    kv = ra.PagedKV(t.k_pool, t.v_pool, torch.as_tensor(w.decode_table(), device=dev))
    lens = torch.as_tensor(w.kv_lens.astype(np.int32), device=dev)
    B, max_kv = w.kv_lens.shape[0], int(w.kv_lens.max())
    out = torch.empty((B, w.Hq, 128), dtype=torch.float32, device=dev)
    ws = torch.empty(ra.decode_workspace_size(B, w.Hq, w.Hkv, max_kv), dtype=torch.uint8,
                     device=dev)
    for _ in range(warmup):
        ra.decode(t.q_decode, kv, lens, max_kv, SCALE, out=out, workspace=ws)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
    for e in ev:
        e[0].record()
        ra.decode(t.q_decode, kv, lens, max_kv, SCALE, out=out, workspace=ws)
        e[1].record()
    torch.cuda.synchronize()
    ms = np.array([e[0].elapsed_time(e[1]) for e in ev])
    nbytes = decode_bytes(w)
    gbs = nbytes / (ms.mean() * 1e-3) / 1e9
    res = {"workload": w.name, "steps": steps, "warmup": warmup,
           "rows": B, "kv_tokens": int(w.kv_lens.sum()),
           "ms": round(float(ms.mean()), 4), "ms_median": round(float(np.median(ms)), 4),
           "ms_min": round(float(ms.min()), 4), "algorithmic_bytes": nbytes,
           "GB_s": round(gbs, 1), "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
           "traffic": measured_traffic("long_decode")}
    del t, kv, out, ws
    torch.cuda.empty_cache()
    return res


def achievable_leg(dev):
    """What this GPU delivers to the kernels, measured now by libra_microbench.so:
    the bf16 matrix-core rate of the append kernel's product on random and on zero
    operands with the shader clock it ran at, LDS read bandwidth, HBM read rates
    (streaming, and shuffled 4 KiB pages as a paged cache is read) and the rate at
    which the L2 feeds the compute units (into LDS and into registers). Context
    for the roofline fractions, which use the published peaks."""
    import torch

    from paper_2603_18815_amd import microbench as mb

    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    res = {"compute_units": cus}
    for name, zeros in (("mfma_bf16_random", False), ("mfma_bf16_zeros", True)):
        tf, ghz = mb.mfma_bf16(2 * cus, 20000, zeros=zeros)
        res[name] = {"TFLOP_s": round(tf, 1), "clock_GHz": round(ghz, 3),
                     "peak_at_clock_TFLOP_s": round(cus * 4096 * ghz / 1e3, 1),
                     "frac_of_published_peak": round(tf / BF16_PEAK_TFLOPS, 4)}
    bpc, ghz, gbs = mb.lds_read(2 * cus, 20000)
    res["lds_read"] = {"GB_s": round(gbs, 0), "clock_GHz": round(ghz, 3),
                       "bytes_per_clock_per_CU": round(gbs / (cus * ghz), 1)}
    # the best of a few occupancies: too few workgroups leave the memory system
    # short of requests, too many crowd it
    for name, paged in (("hbm_read_stream", False), ("hbm_read_paged_4KiB", True)):
        g, per_cu = max((mb.stream_read(4 << 30, paged, k * cus), k) for k in (2, 3, 4, 8))
        res[name] = {"GB_s": round(g, 1), "frac_of_published_peak": round(g / HBM_PEAK_GBS, 4),
                     "workgroups_per_CU": per_cu}
    # the same pass in shuffled 1, 2 and 4 KiB blocks (the size of a 16-token page of one
    # KV head with head dim 128 in fp8 / bf16 is 2 / 4 KiB)
    src = torch.empty(4 << 30, dtype=torch.uint8, device=dev)
    src.fill_(1)
    res["hbm_read_shuffled_blocks_GB_s"] = {
        f"{kb // 1024}KiB": round(max(mb.block_read(src, kb, k * cus) for k in (2, 3, 4)), 1)
        for kb in (1024, 2048, 4096)}
    del src
    torch.cuda.empty_cache()
    # the L2 feeding the compute units (a 2 MiB buffer that stays in every XCD's
    # L2), by direct global-to-LDS loads as the tiled log-prob kernel stages its
    # operands, and by loads into registers; one and two workgroups per CU
    res["l2_read_GB_s"] = {
        name: round(max(mb.l2_read(lds, k * cus, 2000) for k in (1, 2)), 1)
        for name, lds in (("to_lds", True), ("to_registers", False))}
    return res


def mixed_step(ra, synth, dev, steps: int, warmup: int):
    """Time the mixed rollout step of one pool: page write of the step's new
    tokens, append of the append rows, decode of the decode rows (15 % / 85 %
    of B = 512 trajectories, log-normal contexts), on one stream."""
    import torch

    w = synth.config(5)
    t = synth.make_tensors(w, dev)

    def i32(x):
        return torch.as_tensor(np.ascontiguousarray(np.asarray(x, np.int32)), device=dev)

    bt, cu, start = synth.write_plan(w)
    kv_w = ra.PagedKV(t.k_pool, t.v_pool, i32(bt))
    kv_d = kv_w.with_table(i32(w.decode_table()))
    kv_a = kv_w.with_table(i32(w.append_table()))
    cu_t, start_t = i32(cu), i32(start)
    kv_lens, cu_q, ctx = i32(w.kv_lens), i32(w.cu_q()), i32(w.ctx_lens)
    max_kv_d = int(w.kv_lens.max())
    max_q, max_kv_a = int(w.q_lens.max()), int((w.ctx_lens + w.q_lens).max())
    max_new = int(np.diff(cu).max())
    max_pos = int(max(max_kv_d, max_kv_a))
    out_d = torch.empty((w.kv_lens.shape[0], w.Hq, 128), dtype=torch.float32, device=dev)
    out_a = torch.empty((int(w.q_lens.sum()), w.Hq, 128), dtype=torch.float32, device=dev)
    ws = torch.empty(ra.decode_workspace_size(w.kv_lens.shape[0], w.Hq, w.Hkv, max_kv_d),
                     dtype=torch.uint8, device=dev)
    ws_a = torch.empty(ra.append_workspace_size(w.q_lens.shape[0], w.Hq, w.Hkv, max_q),
                       dtype=torch.uint8, device=dev)

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        ra.kv_page_write(t.k_new, t.v_new, cu_t, start_t, kv_w, max_new, max_pos)
        if ev is not None:
            ev[1].record()
        ra.append(t.q_append, cu_q, ctx, kv_a, max_q, max_kv_a, SCALE, out=out_a,
                  workspace=ws_a)
        if ev is not None:
            ev[2].record()
        ra.decode(t.q_decode, kv_d, kv_lens, max_kv_d, SCALE, out=out_d, workspace=ws)
        if ev is not None:
            ev[3].record()

    ws_mix = torch.empty(ra.mixed_workspace_size(w.kv_lens.shape[0], w.q_lens.shape[0], w.Hq,
                                                 w.Hkv, w.Hkv, max_kv_d, max_q),
                         dtype=torch.uint8, device=dev)

    def step_single(ev=None):
        if ev is not None:
            ev[0].record()
        ra.kv_page_write(t.k_new, t.v_new, cu_t, start_t, kv_w, max_new, max_pos)
        if ev is not None:
            ev[1].record()
        ra.mixed(t.q_decode, kv_d, kv_lens, t.q_append, cu_q, ctx, kv_a, max_kv_d, max_q,
                 max_kv_a, SCALE, out_decode=out_d, out_append=out_a, workspace=ws_mix)
        if ev is not None:
            ev[2].record()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    for k in range(steps):
        step(events[k])
    torch.cuda.synchronize()
    for _ in range(warmup):
        step_single()
    torch.cuda.synchronize()
    ev_single = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    for k in range(steps):
        step_single(ev_single[k])
    torch.cuda.synchronize()
    single_ms = np.mean([e[0].elapsed_time(e[2]) for e in ev_single])
    single_attn_ms = np.mean([e[1].elapsed_time(e[2]) for e in ev_single])
    w_ms = np.mean([e[0].elapsed_time(e[1]) for e in events])
    a_ms = np.mean([e[1].elapsed_time(e[2]) for e in events])
    d_ms = np.mean([e[2].elapsed_time(e[3]) for e in events])
    s_ms = np.mean([e[0].elapsed_time(e[3]) for e in events])
    dbytes, aflops = decode_bytes(w), append_flops(w)
    wbytes = write_bytes(int(cu[-1]), w.Hkv)
    # lower bounds at the published peaks: parts in sequence, and perfect overlap
    kv_bytes_app = int((w.ctx_lens.astype(np.int64) + w.q_lens).sum()) * w.Hkv * 128 * 4
    seq_ms = (dbytes + wbytes) / (HBM_PEAK_GBS * 1e6) + aflops / (BF16_PEAK_TFLOPS * 1e9)
    ovl_ms = max((dbytes + wbytes + kv_bytes_app) / (HBM_PEAK_GBS * 1e6),
                 aflops / (BF16_PEAK_TFLOPS * 1e9))
    res = {
        "workload": w.name, "steps": steps, "warmup": warmup,
        "decode_rows": int(w.kv_lens.shape[0]), "append_rows": int(w.q_lens.shape[0]),
        "ms": round(float(s_ms), 4), "page_write_ms": round(float(w_ms), 4),
        "decode_ms": round(float(d_ms), 4), "append_ms": round(float(a_ms), 4),
        "decode_algorithmic_bytes": dbytes, "append_algorithmic_flops": aflops,
        "decode_GB_s": round(dbytes / (d_ms * 1e-3) / 1e9, 1),
        "append_TFLOP_s": round(aflops / (a_ms * 1e-3) / 1e12, 1),
        "bound_sequential_ms": round(seq_ms, 3), "bound_overlap_ms": round(ovl_ms, 3),
        "frac_of_sequential_bound": round(seq_ms / s_ms, 4),
        # decode and append rows in one persistent launch (rollout_attn_mixed)
        "single_launch": {
            "ms": round(float(single_ms), 4),
            "attention_ms": round(float(single_attn_ms), 4),
            "speedup_vs_separate": round(float(s_ms / single_ms), 4),
            "frac_of_sequential_bound": round(seq_ms / single_ms, 4),
            "frac_of_overlap_bound": round(ovl_ms / single_ms, 4),
        },
    }
    del t, out_d, out_a, ws, ws_a, ws_mix
    torch.cuda.empty_cache()
    return res


def shared_prefix_bytes(w) -> int:
    """Algorithmic bytes of shared-prefix decode: each group's shared keys once, each
    row's other keys, q, out, its block-table entries and length."""
    L = w.kv_lens.astype(np.int64)
    D, P = w.head_dim, w.page_size
    pre = np.repeat(w.prefix_len.astype(np.int64), np.diff(w.group_start))
    per_row = ((L - pre) * w.Hkv * D * 4 + w.Hq * D * 2 + w.Hq * D * 4
               + 4 * ((L + P - 1) // P) + 4)
    return int(per_row.sum() + (w.prefix_len.astype(np.int64) * w.Hkv * D * 4).sum())


def shared_prefix_leg(ra, synth, dev, steps: int, warmup: int):
    """Plain decode vs shared-prefix decode of 8 tasks x 8 rollouts (rows of a task
    share its prompt pages)."""
    import torch

    w = synth.config(6)
    t = synth.make_tensors(w, dev)

    def i32(x):
        return torch.as_tensor(np.ascontiguousarray(np.asarray(x, np.int32)), device=dev)

    kv = ra.PagedKV(t.k_pool, t.v_pool, i32(w.decode_table()))
    lens, gs, pre = i32(w.kv_lens), i32(w.group_start), i32(w.prefix_len)
    B, max_kv = w.kv_lens.shape[0], int(w.kv_lens.max())
    mgr, mpl = int(np.diff(w.group_start).max()), int(w.prefix_len.max())
    out = torch.empty((B, w.Hq, 128), dtype=torch.float32, device=dev)
    ws = torch.empty(ra.decode_shared_prefix_workspace_size(B, w.Hq, w.Hkv, max_kv, mpl),
                     dtype=torch.uint8, device=dev)
    # the same rows in an interleaved order (the rollouts of a task 8 rows apart, as
    # requests arrive), for which the cache sees no reuse between a task's rows
    n_g = w.group_start.size - 1
    perm = np.arange(B).reshape(n_g, -1).T.reshape(-1)
    kv_i = ra.PagedKV(t.k_pool, t.v_pool, i32(w.decode_table()[perm]))
    q_i, lens_i = t.q_decode[torch.as_tensor(perm, device=dev)].contiguous(), i32(w.kv_lens[perm])
    calls = {
        "plain": lambda: ra.decode(t.q_decode, kv, lens, max_kv, SCALE, out=out, workspace=ws),
        "plain_interleaved": lambda: ra.decode(q_i, kv_i, lens_i, max_kv, SCALE, out=out,
                                               workspace=ws),
        "shared": lambda: ra.decode_shared_prefix(t.q_decode, kv, lens, gs, pre, mgr, mpl,
                                                  max_kv, SCALE, out=out, workspace=ws),
    }
    ms = {}
    for name, fn in calls.items():
        for _ in range(warmup):
            fn()
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
        for e in ev:
            e[0].record()
            fn()
            e[1].record()
        torch.cuda.synchronize()
        ms[name] = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    plain_b, shared_b = decode_bytes(w), shared_prefix_bytes(w)
    res = {
        "workload": w.name, "steps": steps, "warmup": warmup,
        "plain_ms": round(ms["plain"], 4),
        "plain_interleaved_ms": round(ms["plain_interleaved"], 4),
        "shared_ms": round(ms["shared"], 4),
        "speedup_vs_plain": round(ms["plain"] / ms["shared"], 3),
        "speedup_vs_plain_interleaved": round(ms["plain_interleaved"] / ms["shared"], 3),
        "plain_algorithmic_bytes": plain_b, "shared_algorithmic_bytes": shared_b,
        "plain_GB_s": round(plain_b / (ms["plain"] * 1e-3) / 1e9, 1),
        "plain_interleaved_GB_s": round(plain_b / (ms["plain_interleaved"] * 1e-3) / 1e9, 1),
        "shared_GB_s": round(shared_b / (ms["shared"] * 1e-3) / 1e9, 1),
        "shared_frac_hbm_peak": round(shared_b / (ms["shared"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "shared_effective_GB_s": round(plain_b / (ms["shared"] * 1e-3) / 1e9, 1),
    }
    del t, out, ws, q_i
    torch.cuda.empty_cache()
    return res


def fp8_decode_bytes(w) -> int:
    """Algorithmic bytes of decode over fp8 pools: as decode_bytes with one byte per
    K/V element."""
    L = w.kv_lens.astype(np.int64)
    D, P = w.head_dim, w.page_size
    per_row = L * w.Hkv * D * 2 + w.Hq * D * 2 + w.Hq * D * 4 + 4 * ((L + P - 1) // P) + 4
    return int(per_row.sum())


def fp8_kv_leg(ra, synth, dev, wd, td, wa, ta, steps: int, warmup: int):
    """Decode of the B = 64 decode workload, and append of the B = 32 append workload,
    over fp8 (E4M3) pools beside the same rows over the bf16 pools, each timed alone."""
    import torch

    def i32(x):
        return torch.as_tensor(np.ascontiguousarray(np.asarray(x, np.int32)), device=dev)

    ks = vs = 2.0 ** -5
    gen = synth.value_generator(1234, dev)
    n = wd.layout.num_pages
    k8 = synth.randn_fp8_codes((n, wd.Hkv, 16, 128), gen, dev, ks)
    v8 = synth.randn_fp8_codes((n, wd.Hkv, 128, 16), gen, dev, vs)
    bt = i32(wd.decode_table())
    kv8 = ra.PagedKV(k8, v8, bt, ks, vs)
    kv16 = ra.PagedKV(td.k_pool, td.v_pool, bt)
    lens, max_kv, B = i32(wd.kv_lens), int(wd.kv_lens.max()), wd.kv_lens.shape[0]
    out = torch.empty((B, wd.Hq, 128), dtype=torch.float32, device=dev)
    ws = torch.empty(ra.decode_workspace_size(B, wd.Hq, wd.Hkv, max_kv), dtype=torch.uint8,
                     device=dev)
    na = wa.layout.num_pages
    ka8 = synth.randn_fp8_codes((na, wa.Hkv, 16, 128), gen, dev, ks)
    va8 = synth.randn_fp8_codes((na, wa.Hkv, 128, 16), gen, dev, vs)
    bta = i32(wa.append_table())
    kva8 = ra.PagedKV(ka8, va8, bta, ks, vs)
    kva16 = ra.PagedKV(ta.k_pool, ta.v_pool, bta)
    cu_q, ctx = i32(wa.cu_q()), i32(wa.ctx_lens)
    max_q, max_kva = int(wa.q_lens.max()), int((wa.ctx_lens + wa.q_lens).max())
    out_a = torch.empty((int(wa.q_lens.sum()), wa.Hq, 128), dtype=torch.float32, device=dev)
    ws_a = torch.empty(ra.append_workspace_size(wa.q_lens.shape[0], wa.Hq, wa.Hkv, max_q),
                       dtype=torch.uint8, device=dev)
    ms = {}
    calls = [("bf16", lambda: ra.decode(td.q_decode, kv16, lens, max_kv, SCALE, out=out,
                                        workspace=ws)),
             ("fp8", lambda: ra.decode(td.q_decode, kv8, lens, max_kv, SCALE, out=out,
                                       workspace=ws)),
             ("append_bf16", lambda: ra.append(ta.q_append, cu_q, ctx, kva16, max_q, max_kva,
                                               SCALE, out=out_a, workspace=ws_a)),
             ("append_fp8", lambda: ra.append(ta.q_append, cu_q, ctx, kva8, max_q, max_kva,
                                              SCALE, out=out_a, workspace=ws_a))]
    for name, fn in calls:
        for _ in range(warmup):
            fn()
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
        for e in ev:
            e[0].record()
            fn()
            e[1].record()
        torch.cuda.synchronize()
        ms[name] = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    b16, b8 = decode_bytes(wd), fp8_decode_bytes(wd)
    res = {
        "workload": wd.name + ", fp8 E4M3 pool (per-pool scales)",
        "steps": steps, "warmup": warmup,
        "bf16_ms": round(ms["bf16"], 4), "fp8_ms": round(ms["fp8"], 4),
        "speedup": round(ms["bf16"] / ms["fp8"], 3),
        "fp8_algorithmic_bytes": b8,
        "fp8_GB_s": round(b8 / (ms["fp8"] * 1e-3) / 1e9, 1),
        "fp8_frac_hbm_peak": round(b8 / (ms["fp8"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "bf16_GB_s": round(b16 / (ms["bf16"] * 1e-3) / 1e9, 1),
        "append_workload": wa.name,
        "append_bf16_ms": round(ms["append_bf16"], 4),
        "append_fp8_ms": round(ms["append_fp8"], 4),
        "append_fp8_TFLOP_s": round(append_flops(wa) / (ms["append_fp8"] * 1e-3) / 1e12, 1),
    }
    del k8, v8, out, ws, ka8, va8, out_a, ws_a
    torch.cuda.empty_cache()
    return res


def append_write_leg(ra, dev, wa, ta, kv_aw, kv_a, steps: int, warmup: int):
    """The append workload's page write + append as two calls and as one fused call
    (rollout_attn_append_write), each timed alone; and the same with rotary
    position embedding on write (Qwen3's table: theta 1e6), as two calls
    (kv_page_write_rope + append) and fused (rollout_attn_append_write_rope)."""
    import torch

    def i32(x):
        return torch.as_tensor(np.ascontiguousarray(np.asarray(x, np.int32)), device=dev)

    cu_q, ctx = i32(wa.cu_q()), i32(wa.ctx_lens)
    max_q, max_kv = int(wa.q_lens.max()), int((wa.ctx_lens + wa.q_lens).max())
    n = int(wa.q_lens.sum())
    k_new, v_new = ta.k_new[-n:], ta.v_new[-n:]
    out = torch.empty((n, wa.Hq, 128), dtype=torch.float32, device=dev)
    ws = torch.empty(ra.append_workspace_size(wa.q_lens.shape[0], wa.Hq, wa.Hkv, max_q),
                     dtype=torch.uint8, device=dev)
    inv = 1e6 ** (-2.0 * np.arange(64) / 128.0)
    ang = np.arange(max_kv, dtype=np.float64)[:, None] * inv[None, :]
    table = torch.from_numpy(np.concatenate([np.cos(ang), np.sin(ang)], 1).astype(np.float32))
    table = table.to(dev)
    calls = {
        "separate": lambda: (ra.kv_page_write(k_new, v_new, cu_q, ctx, kv_aw, max_q, max_kv),
                             ra.append(ta.q_append, cu_q, ctx, kv_a, max_q, max_kv, SCALE,
                                       out=out, workspace=ws)),
        "fused": lambda: ra.append_write(ta.q_append, k_new, v_new, cu_q, ctx, kv_a, max_q,
                                         max_kv, SCALE, out=out, workspace=ws),
        "rope_write": lambda: ra.kv_page_write(k_new, v_new, cu_q, ctx, kv_aw, max_q, max_kv,
                                               cos_sin=table),
        "rope_fused": lambda: ra.append_write(ta.q_append, k_new, v_new, cu_q, ctx, kv_a, max_q,
                                              max_kv, SCALE, out=out, workspace=ws,
                                              cos_sin=table),
    }
    ms = {}
    for name, fn in calls.items():
        for _ in range(warmup):
            fn()
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
        for e in ev:
            e[0].record()
            fn()
            e[1].record()
        torch.cuda.synchronize()
        ms[name] = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    flops = append_flops(wa)
    res = {"workload": wa.name, "steps": steps, "warmup": warmup,
           "separate_ms": round(ms["separate"], 4), "fused_ms": round(ms["fused"], 4),
           "speedup": round(ms["separate"] / ms["fused"], 4),
           "fused_TFLOP_s": round(flops / (ms["fused"] * 1e-3) / 1e12, 1),
           "rope_write_ms": round(ms["rope_write"], 4),
           "rope_fused_ms": round(ms["rope_fused"], 4),
           "rope_fused_TFLOP_s": round(flops / (ms["rope_fused"] * 1e-3) / 1e12, 1)}
    del out, ws, table
    return res


def logprob_leg(ra, synth, dev, steps: int, warmup: int):
    """token_logprob on the Qwen3-8B LM head (V = 151936, D = 4096): a decode
    batch of 64 tokens (bound by reading W) and 1024 tokens (bound by the
    products), with W row-major and packed (token_logprob_packed; the one-time
    packing is timed on its own)."""
    import torch

    V, D = 151936, 4096
    gen = synth.value_generator(7, dev)
    W = (synth.randn_bf16((V, D), gen, dev).float() * (1.0 / math.sqrt(D))).to(torch.bfloat16)
    Wp = ra.token_logprob_pack_weight(W)
    res = {"workload": f"token log-probabilities, LM head V={V} D={D} (Qwen3-8B), bf16"}

    def timed(fn):
        for _ in range(warmup):
            fn()
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
        for e in ev:
            e[0].record()
            fn()
            e[1].record()
        torch.cuda.synchronize()
        return float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))

    res["pack_ms"] = round(timed(lambda: ra.token_logprob_pack_weight(W, out=Wp)), 4)
    for N in (64, 1024):
        h = synth.randn_bf16((N, D), gen, dev)
        t = torch.randint(0, V, (N,), dtype=torch.int32, device=dev, generator=gen)
        out = torch.empty(N, dtype=torch.float32, device=dev)
        ws = torch.empty(ra.token_logprob_workspace_size(N, V, D), dtype=torch.uint8, device=dev)
        nbytes = V * D * 2 + N * D * 2 + N * 8
        flops = 2 * N * V * D
        for key, fn in ((f"N{N}", lambda: ra.token_logprob(h, W, t, 1.0, out=out, workspace=ws)),
                        (f"N{N}_packed", lambda: ra.token_logprob_packed(
                            h, Wp, V, t, 1.0, out=out, workspace=ws))):
            ms = timed(fn)
            gbs, tfs = nbytes / (ms * 1e-3) / 1e9, flops / (ms * 1e-3) / 1e12
            res[key] = {"ms": round(ms, 4), "algorithmic_bytes": nbytes,
                        "algorithmic_flops": flops, "GB_s": round(gbs, 1),
                        "TFLOP_s": round(tfs, 1),
                        "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
                        "frac_bf16_peak": round(tfs / BF16_PEAK_TFLOPS, 4)}
        del h, t, out, ws
    del W, Wp
    torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--cpu-seconds", type=float, default=8.0,
                    help="time budget of each leg (decode, append) of the CPU oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-shared-prefix", action="store_true",
                    help="skip the shared-prefix decode leg (8 tasks x 8 rollouts)")
    ap.add_argument("--no-append-write", action="store_true",
                    help="skip the fused page write + append leg")
    ap.add_argument("--no-fp8", action="store_true",
                    help="skip the fp8 KV pool decode leg")
    ap.add_argument("--no-logprob", action="store_true",
                    help="skip the token log-probability leg (Qwen3-8B LM head)")
    ap.add_argument("--no-mixed", action="store_true",
                    help="skip the mixed-step leg (B = 512, 85 %% decode / 15 %% append rows)")
    ap.add_argument("--no-long-decode", action="store_true",
                    help="skip the long-horizon decode leg (B = 256, Hq = 64)")
    ap.add_argument("--no-achievable", action="store_true",
                    help="skip the hardware-ceiling microbenchmarks")
    ap.add_argument("--only", choices=["write", "decode", "append", "copy", "mixed", "logprob",
                                       "decode_fp8", "append_fp8", "long_decode", "mfma",
                                       "stream"],
                    help="run only this part of the step --steps times after --warmup "
                         "(for rocprofv3 runs; 'copy' is a 1 GiB torch copy used to "
                         "calibrate the HBM byte counters, 'mixed' the mixed-step leg, "
                         "'logprob' the LM-head log-probability leg, 'decode_fp8' / 'append_fp8' "
                         "the decode / append workload over fp8 pools, 'long_decode' the "
                         "long-horizon decode, 'mfma' / 'stream' the matrix-core and HBM-read "
                         "microbenchmarks); prints no JSON line")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(rows shard by trajectory with no exchange; see the design notes).",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2603_18815_amd as ra
    import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.only == "mixed":
        res = mixed_step(ra, synth, dev, args.steps, args.warmup)
        print(f"[bench] mixed step {json.dumps(res)}", flush=True)
        return
    if args.only == "logprob":
        res = logprob_leg(ra, synth, dev, args.steps, args.warmup)
        print(f"[bench] token_logprob {json.dumps(res)}", flush=True)
        return
    if args.only == "long_decode":
        res = long_decode_leg(ra, synth, dev, args.steps, args.warmup)
        print(f"[bench] long decode {json.dumps(res)}", flush=True)
        return
    if args.only in ("mfma", "stream"):
        from paper_2603_18815_amd import microbench as mb
        cus = torch.cuda.get_device_properties(dev).multi_processor_count
        for _ in range(args.warmup + args.steps):
            if args.only == "mfma":
                tf, ghz = mb.mfma_bf16(2 * cus, 20000, reps=1)
            else:
                g = mb.stream_read(4 << 30, True, 3 * cus, reps=1)
        print(f"[bench] ran {args.only} {args.warmup} + {args.steps} times", flush=True)
        return
    wd, wa = synth.config(2), synth.config(3)
    td, ta = synth.make_tensors(wd, dev), synth.make_tensors(wa, dev)

    def i32(x):
        return torch.as_tensor(np.ascontiguousarray(np.asarray(x, np.int32)), device=dev)

    # decode workload: the decode token of each row is written at kv_len - 1
    bt_d, cu_d, st_d = synth.write_plan(wd)
    bt_a, cu_a, st_a = synth.write_plan(wa)
    kv_d = ra.PagedKV(td.k_pool, td.v_pool, i32(wd.decode_table()))
    kv_a = ra.PagedKV(ta.k_pool, ta.v_pool, i32(wa.append_table()))
    kv_dw = kv_d.with_table(i32(bt_d))
    kv_aw = kv_a.with_table(i32(bt_a))
    cu_d_t, st_d_t, cu_a_t, st_a_t = i32(cu_d), i32(st_d), i32(cu_a), i32(st_a)
    kv_lens = i32(wd.kv_lens)
    cu_q, ctx = i32(wa.cu_q()), i32(wa.ctx_lens)
    max_kv_d = int(wd.kv_lens.max())
    max_q, max_kv_a = int(wa.q_lens.max()), int((wa.ctx_lens + wa.q_lens).max())
    out_d = torch.empty((wd.kv_lens.shape[0], wd.Hq, 128), dtype=torch.float32, device=dev)
    out_a = torch.empty((int(wa.q_lens.sum()), wa.Hq, 128), dtype=torch.float32, device=dev)
    ws = torch.empty(ra.decode_workspace_size(wd.kv_lens.shape[0], wd.Hq, wd.Hkv, max_kv_d),
                     dtype=torch.uint8, device=dev)
    ws_a = torch.empty(ra.append_workspace_size(wa.q_lens.shape[0], wa.Hq, wa.Hkv, max_q),
                       dtype=torch.uint8, device=dev)
    max_new_d, max_pos_d = 1, max_kv_d
    max_new_a, max_pos_a = max_q, max_kv_a

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        ra.kv_page_write(td.k_new, td.v_new, cu_d_t, st_d_t, kv_dw, max_new_d, max_pos_d)
        ra.kv_page_write(ta.k_new, ta.v_new, cu_a_t, st_a_t, kv_aw, max_new_a, max_pos_a)
        if ev is not None:
            ev[1].record()
        ra.append(ta.q_append, cu_q, ctx, kv_a, max_q, max_kv_a, SCALE, out=out_a,
                  workspace=ws_a)
        if ev is not None:
            ev[2].record()
        ra.decode(td.q_decode, kv_d, kv_lens, max_kv_d, SCALE, out=out_d, workspace=ws)
        if ev is not None:
            ev[3].record()

    if args.only:
        if args.only == "copy":
            src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
            dst = torch.empty_like(src)
            src.fill_(1)
            part = lambda: dst.copy_(src)
        elif args.only == "decode_fp8":
            # the fp8 pools of the fp8 leg (same seed and scales), the decode workload's rows
            ks = vs = 2.0 ** -5
            gen = synth.value_generator(1234, dev)
            n = wd.layout.num_pages
            kv8 = ra.PagedKV(synth.randn_fp8_codes((n, wd.Hkv, 16, 128), gen, dev, ks),
                             synth.randn_fp8_codes((n, wd.Hkv, 128, 16), gen, dev, vs),
                             i32(wd.decode_table()), ks, vs)
            part = lambda: ra.decode(td.q_decode, kv8, kv_lens, max_kv_d, SCALE, out=out_d,
                                     workspace=ws)
        elif args.only == "append_fp8":
            # fp8 pools for the append workload's rows (scales as in the fp8 leg)
            ks = vs = 2.0 ** -5
            gen = synth.value_generator(1235, dev)
            n = wa.layout.num_pages
            kva8 = ra.PagedKV(synth.randn_fp8_codes((n, wa.Hkv, 16, 128), gen, dev, ks),
                              synth.randn_fp8_codes((n, wa.Hkv, 128, 16), gen, dev, vs),
                              i32(wa.append_table()), ks, vs)
            part = lambda: ra.append(ta.q_append, cu_q, ctx, kva8, max_q, max_kv_a, SCALE,
                                     out=out_a, workspace=ws_a)
        else:
            part = {"write": lambda: (ra.kv_page_write(td.k_new, td.v_new, cu_d_t, st_d_t, kv_dw,
                                                       max_new_d, max_pos_d),
                                      ra.kv_page_write(ta.k_new, ta.v_new, cu_a_t, st_a_t, kv_aw,
                                                       max_new_a, max_pos_a)),
                    "decode": lambda: ra.decode(td.q_decode, kv_d, kv_lens, max_kv_d, SCALE,
                                                out=out_d, workspace=ws),
                    "append": lambda: ra.append(ta.q_append, cu_q, ctx, kv_a, max_q, max_kv_a,
                                                SCALE, out=out_a, workspace=ws_a)}[args.only]
        for _ in range(args.warmup + args.steps):
            part()
        torch.cuda.synchronize()
        print(f"[bench] ran {args.only} {args.warmup} + {args.steps} times", flush=True)
        return

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(events[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    w_ms = np.array([e[0].elapsed_time(e[1]) for e in events])
    a_ms = np.array([e[1].elapsed_time(e[2]) for e in events])
    d_ms = np.array([e[2].elapsed_time(e[3]) for e in events])
    step_ms = np.array([e[0].elapsed_time(e[3]) for e in events])

    dbytes = decode_bytes(wd)
    aflops = append_flops(wa)
    n_new = int(cu_d[-1] + cu_a[-1])
    wbytes = write_bytes(n_new, wd.Hkv)
    dec_gbs = dbytes / (d_ms.mean() * 1e-3) / 1e9
    app_tfs = aflops / (a_ms.mean() * 1e-3) / 1e12

    shared = None
    if not args.no_shared_prefix:
        shared = shared_prefix_leg(ra, synth, dev, args.steps, args.warmup)
    append_write = None
    if not args.no_append_write:
        append_write = append_write_leg(ra, dev, wa, ta, kv_aw, kv_a, args.steps, args.warmup)
    fp8 = None
    if not args.no_fp8:
        fp8 = fp8_kv_leg(ra, synth, dev, wd, td, wa, ta, args.steps, args.warmup)
    logprob = None
    if not args.no_logprob:
        logprob = logprob_leg(ra, synth, dev, args.steps, args.warmup)
    mixed = None
    if not args.no_mixed:
        mixed = mixed_step(ra, synth, dev, min(args.steps, 10), min(args.warmup, 2))
    long_decode = None
    if not args.no_long_decode:
        long_decode = long_decode_leg(ra, synth, dev, args.steps, args.warmup)
    achievable = None
    if not args.no_achievable:
        achievable = achievable_leg(dev)

    cpu_dec = cpu_app = cpu_single = cpu_long = None
    if not args.no_cpu_baseline:
        cpu_dec, cpu_app, cpu_single, cpu_long = cpu_baseline(wd, td, wa, ta, args.cpu_seconds)

    rec = {
        "metric": "decode attn HBM GB/s (% of peak) + append TFLOP/s, Qwen3-8B GQA shape",
        "value": round(dec_gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(float(step_ms.mean()), 4),
        "wall_ms_per_step": round(wall * 1e3 / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; bf16 N(0,1) K/V/q, shuffled 16-token pages)",
        "config": {
            "workload": "rollout attention step, Qwen3-8B GQA (Hq=32, Hkv=8, d=128, page 16): "
                        "page write + append B=32 ctx~U[2048,24576] T~U[64,2048] + "
                        "decode B=64 L~U[4096,32768]",
            "decode_rows": int(wd.kv_lens.shape[0]),
            "decode_kv_tokens": int(wd.kv_lens.sum()),
            "append_rows": int(wa.q_lens.shape[0]),
            "append_q_tokens": int(wa.q_lens.sum()),
            "append_ctx_tokens": int(wa.ctx_lens.sum()),
            "new_tokens_written": n_new,
            "parallelism": "1 GPU",
        },
        "decode": {"ms": round(float(d_ms.mean()), 4), "ms_median": round(float(np.median(d_ms)), 4),
                   "ms_min": round(float(d_ms.min()), 4),
                   "algorithmic_bytes": dbytes, "GB_s": round(dec_gbs, 1),
                   "frac_hbm_peak": round(dec_gbs / HBM_PEAK_GBS, 4)},
        "append": {"ms": round(float(a_ms.mean()), 4), "ms_median": round(float(np.median(a_ms)), 4),
                   "ms_min": round(float(a_ms.min()), 4),
                   "algorithmic_flops": aflops, "TFLOP_s": round(app_tfs, 1),
                   "frac_bf16_peak": round(app_tfs / BF16_PEAK_TFLOPS, 4)},
        "page_write": {"ms": round(float(w_ms.mean()), 4), "algorithmic_bytes": wbytes,
                       "GB_s": round(wbytes / (w_ms.mean() * 1e-3) / 1e9, 1)},
        "roofline": {"kernel": "rollout_attn_decode (decode_split_kernel + decode_combine_kernel)",
                     "bound": "hbm", "achieved": round(dec_gbs, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(dec_gbs / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic("decode")},
        "roofline_append": {"kernel": "rollout_attn_append (mixed_plan_kernel + mixed_kernel)",
                            "bound": "mfma",
                            "achieved": round(app_tfs, 1), "peak": BF16_PEAK_TFLOPS,
                            "unit": "TFLOP/s", "frac": round(app_tfs / BF16_PEAK_TFLOPS, 4),
                            "traffic": measured_traffic("append")},
        "mixed_step": mixed,
        "shared_prefix_decode": shared,
        "append_write": append_write,
        "fp8_kv_decode": fp8,
        "token_logprob": logprob,
        "long_horizon_decode": long_decode,
        "achievable": achievable,
        "paper_context": {
            "note": "the paper's own system-level rollout throughput, on its hardware; context "
                    "only, not comparable to the kernel metric (the paper publishes no kernel "
                    "number)",
            "metric": "rollout throughput, full system (Table 3)", "value": 0.37,
            "unit": "instances/s", "hardware": "8x NVIDIA H100", "model": "Qwen3-14B",
            "workload": "DAPO RL on SWE tasks"},
        "cpu_baseline": cpu_dec,
        "cpu_baseline_append": cpu_app,
        "cpu_baseline_single_thread": cpu_single,
        "cpu_baseline_long_decode": cpu_long,
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
