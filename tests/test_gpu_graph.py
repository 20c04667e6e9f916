"""The library's calls under HIP graph capture (through the C ABI).

Serving loops capture a whole step into a graph and replay it. Every entry
point allocates nothing, never synchronizes and clears its own work counters
with a kernel, so a captured step must replay to the same results as the
eager calls, every time. The graph here holds one rollout step (page write,
append, decode), the fused write + append and the single-launch mixed step;
it is replayed several times with eager work and synchronizations between the
replays, and every replay is compared bitwise with the eager results. A second
graph holds the fp8-pool step with keys rotated on write, the fused rotated
write + append, and the LM-head log-probabilities (row-major and packed).
"""
import math

import numpy as np
import pytest
import torch

import paper_2603_18815_amd as ra
import synth

pytestmark = pytest.mark.gpu
SCALE = 1.0 / math.sqrt(128)


def i32(x, dev):
    return torch.as_tensor(np.ascontiguousarray(np.asarray(x, np.int32)), device=dev)


def say(msg):
    print(f"[gpu-test] {msg}", flush=True)


def replay_and_check(step, outs, names, pools):
    """Eager step, then a captured one replayed four times; every replay must
    equal the eager results bit for bit and leave the pools as they were."""
    step()                                   # eager: also brings the pools to their end state
    torch.cuda.synchronize()
    ref = [o.clone() for o in outs]
    pools0 = [p.clone() for p in pools]
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()                               # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        step()
    for rep in range(4):
        for o in outs:
            o.fill_(float("nan"))            # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for name, o, r in zip(names, outs, ref):
            assert torch.equal(o, r), f"replay {rep}: {name} differs from the eager result"
        for p, p0 in zip(pools, pools0):
            assert torch.equal(p, p0), f"replay {rep}: pool changed"
        say(f"graph replay {rep}: bitwise equal to eager")


def test_step_replays_in_a_graph(device):
    w = synth.mixed_workload(41, 24, 32, 8, 0.35,
                             lambda r, n: synth.uniform_int(r, n, 0, 1500),
                             lambda r, n: synth.uniform_int(r, n, 1, 300),
                             "graph step")
    say(f"graph: {w.decode_rows.size} decode rows, {w.append_rows.size} append rows")
    t = synth.make_tensors(w, device)
    kd = ra.PagedKV(t.k_pool, t.v_pool, i32(w.decode_table(), device))
    ka = ra.PagedKV(t.k_pool, t.v_pool, i32(w.append_table(), device))
    bt_w, cu_w, st_w = synth.write_plan(w)
    kw = kd.with_table(i32(bt_w, device))
    cu_w_t, st_w_t = i32(cu_w, device), i32(st_w, device)
    lens = i32(w.kv_lens, device)
    cu_q, ctx = i32(w.cu_q(), device), i32(w.ctx_lens, device)
    Bd, Ba = w.kv_lens.size, w.q_lens.size
    mk, mq = int(w.kv_lens.max()), int(w.q_lens.max())
    mka = int((w.ctx_lens + w.q_lens).max())
    max_new, max_pos = int(np.diff(cu_w).max()), int((np.diff(cu_w) + st_w).max())
    nq = int(w.q_lens.sum())
    k_chunk, v_chunk = t.k_new[-nq:], t.v_new[-nq:]
    f32 = dict(dtype=torch.float32, device=device)
    out_d, lse_d = torch.empty((Bd, w.Hq, 128), **f32), torch.empty((Bd, w.Hq), **f32)
    out_a, lse_a = torch.empty((nq, w.Hq, 128), **f32), torch.empty((nq, w.Hq), **f32)
    out_f = torch.empty((nq, w.Hq, 128), **f32)
    out_md, out_ma = torch.empty((Bd, w.Hq, 128), **f32), torch.empty((nq, w.Hq, 128), **f32)
    u8 = dict(dtype=torch.uint8, device=device)
    ws_d = torch.empty(ra.decode_workspace_size(Bd, w.Hq, w.Hkv, mk), **u8)
    ws_a = torch.empty(ra.append_workspace_size(Ba, w.Hq, w.Hkv, mq), **u8)
    ws_f = torch.empty(ra.append_workspace_size(Ba, w.Hq, w.Hkv, mq), **u8)
    ws_m = torch.empty(ra.mixed_workspace_size(Bd, Ba, w.Hq, w.Hkv, w.Hkv, mk, mq), **u8)

    def step():
        ra.kv_page_write(t.k_new, t.v_new, cu_w_t, st_w_t, kw, max_new, max_pos)
        ra.append(t.q_append, cu_q, ctx, ka, mq, mka, SCALE, out=out_a, lse=lse_a,
                  workspace=ws_a)
        ra.decode(t.q_decode, kd, lens, mk, SCALE, out=out_d, lse=lse_d, workspace=ws_d)
        ra.append_write(t.q_append, k_chunk, v_chunk, cu_q, ctx, ka, mq, mka, SCALE, out=out_f,
                        workspace=ws_f)
        ra.mixed(t.q_decode, kd, lens, t.q_append, cu_q, ctx, ka, mk, mq, mka, SCALE,
                 out_decode=out_md, out_append=out_ma, workspace=ws_m)

    outs = (out_d, lse_d, out_a, lse_a, out_f, out_md, out_ma)
    replay_and_check(step, outs, ("decode", "decode lse", "append", "append lse", "append_write",
                                  "mixed decode", "mixed append"), (t.k_pool, t.v_pool))


def rope_table(theta, rows):
    """cos | sin of p * theta^(-2i/128) for p < rows (fp64 math, stored fp32)."""
    inv = float(theta) ** (-2.0 * np.arange(64) / 128.0)
    ang = np.arange(rows, dtype=np.float64)[:, None] * inv[None, :]
    return np.concatenate([np.cos(ang), np.sin(ang)], axis=1).astype(np.float32)


def test_fp8_rope_logprob_step_replays_in_a_graph(device):
    w = synth.mixed_workload(43, 20, 32, 8, 0.4,
                             lambda r, n: synth.uniform_int(r, n, 1, 1200),
                             lambda r, n: synth.uniform_int(r, n, 1, 200),
                             "graph fp8 rope step")
    say(f"graph fp8/rope: {w.decode_rows.size} decode rows, {w.append_rows.size} append rows")
    gen = synth.value_generator(43, device)
    ks, vs = 0.05, 0.04
    n_pages, Hkv = w.layout.num_pages, w.Hkv
    k_pool = synth.randn_fp8_codes((n_pages, Hkv, 16, 128), gen, device, ks)
    v_pool = synth.randn_fp8_codes((n_pages, Hkv, 128, 16), gen, device, vs)
    t = synth.make_tensors(w, device, gen)
    kd = ra.PagedKV(k_pool, v_pool, i32(w.decode_table(), device), ks, vs)
    ka = kd.with_table(i32(w.append_table(), device))
    bt_w, cu_w, st_w = synth.write_plan(w)
    kw = kd.with_table(i32(bt_w, device))
    cu_w_t, st_w_t = i32(cu_w, device), i32(st_w, device)
    lens = i32(w.kv_lens, device)
    cu_q, ctx = i32(w.cu_q(), device), i32(w.ctx_lens, device)
    Bd, Ba = w.kv_lens.size, w.q_lens.size
    mk, mq = int(w.kv_lens.max()), int(w.q_lens.max())
    mka = int((w.ctx_lens + w.q_lens).max())
    max_new, max_pos = int(np.diff(cu_w).max()), int((np.diff(cu_w) + st_w).max())
    tab = torch.from_numpy(rope_table(1e6, max(max_pos, mka) + 3)).to(device)
    nq = int(w.q_lens.sum())
    k_chunk, v_chunk = t.k_new[-nq:], t.v_new[-nq:]
    # LM head: V = 1000 (not a multiple of the 128-row packing), D = 128
    V, N = 1000, 48
    W = synth.randn_bf16((V, 128), gen, device)
    h = synth.randn_bf16((N, 128), gen, device)
    targets = i32(np.random.default_rng(43).integers(0, V, N), device)
    Wp = ra.token_logprob_pack_weight(W)
    f32 = dict(dtype=torch.float32, device=device)
    u8 = dict(dtype=torch.uint8, device=device)
    out_d, lse_d = torch.empty((Bd, w.Hq, 128), **f32), torch.empty((Bd, w.Hq), **f32)
    out_f, lse_f = torch.empty((nq, w.Hq, 128), **f32), torch.empty((nq, w.Hq), **f32)
    out_md, out_ma = torch.empty((Bd, w.Hq, 128), **f32), torch.empty((nq, w.Hq, 128), **f32)
    lp, lp_lse = torch.empty((N,), **f32), torch.empty((N,), **f32)
    lpp, lpp_lse = torch.empty((N,), **f32), torch.empty((N,), **f32)
    ws_d = torch.empty(ra.decode_workspace_size(Bd, w.Hq, Hkv, mk), **u8)
    ws_f = torch.empty(ra.append_workspace_size(Ba, w.Hq, Hkv, mq), **u8)
    ws_m = torch.empty(ra.mixed_workspace_size(Bd, Ba, w.Hq, Hkv, Hkv, mk, mq), **u8)
    ws_l = torch.empty(ra.token_logprob_workspace_size(N, V, 128), **u8)
    ws_p = torch.empty(ra.token_logprob_workspace_size(N, V, 128), **u8)

    def step():
        ra.kv_page_write(t.k_new, t.v_new, cu_w_t, st_w_t, kw, max_new, max_pos, cos_sin=tab)
        ra.append_write(t.q_append, k_chunk, v_chunk, cu_q, ctx, ka, mq, mka, SCALE, out=out_f,
                        lse=lse_f, workspace=ws_f, cos_sin=tab)
        ra.decode(t.q_decode, kd, lens, mk, SCALE, out=out_d, lse=lse_d, workspace=ws_d)
        ra.mixed(t.q_decode, kd, lens, t.q_append, cu_q, ctx, ka, mk, mq, mka, SCALE,
                 out_decode=out_md, out_append=out_ma, workspace=ws_m)
        ra.token_logprob(h, W, targets, out=lp, lse=lp_lse, workspace=ws_l)
        ra.token_logprob_packed(h, Wp, V, targets, out=lpp, lse=lpp_lse, workspace=ws_p)

    outs = (out_d, lse_d, out_f, lse_f, out_md, out_ma, lp, lp_lse, lpp, lpp_lse)
    replay_and_check(step, outs, ("fp8 decode", "fp8 decode lse", "rope append_write",
                                  "rope append_write lse", "fp8 mixed decode",
                                  "fp8 mixed append", "logprob", "logprob lse",
                                  "packed logprob", "packed logprob lse"), (k_pool, v_pool))


def test_shared_prefix_and_large_batch_logprob_replay_in_a_graph(device):
    """Shared-prefix decode (prefix and row items in one launch) and the
    log-probabilities of a batch large enough for the tiled LM-head kernel
    (N >= 512), captured together."""
    rng = np.random.default_rng(47)
    sizes, Hq, Hkv = [5, 8, 3], 32, 8
    pre = np.array([40, 9, 70], np.int64) * 16
    suffix = rng.integers(1, 900, size=sum(sizes))
    lay = synth.shared_prefix_layout(rng, sizes, pre, suffix)
    say(f"graph shared prefix groups={sizes} + logprob N=600")
    gen = synth.value_generator(47, device)
    k_pool = synth.randn_bf16((lay.num_pages, Hkv, 16, 128), gen, device)
    v_pool = synth.randn_bf16((lay.num_pages, Hkv, 128, 16), gen, device)
    q = synth.randn_bf16((len(suffix), Hq, 128), gen, device)
    kv = ra.PagedKV(k_pool, v_pool, i32(lay.block_table, device))
    lens = lay.row_tokens.astype(np.int32)
    gs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    lens_t, gs_t, pre_t = i32(lens, device), i32(gs, device), i32(pre, device)
    B, mk, mg, mp = len(suffix), int(lens.max()), max(sizes), int(pre.max())
    V, N, D = 1000, 600, 128
    W = synth.randn_bf16((V, D), gen, device)
    h = synth.randn_bf16((N, D), gen, device)
    targets = i32(np.random.default_rng(48).integers(0, V, N), device)
    Wp = ra.token_logprob_pack_weight(W)
    f32 = dict(dtype=torch.float32, device=device)
    u8 = dict(dtype=torch.uint8, device=device)
    out, lse = torch.empty((B, Hq, 128), **f32), torch.empty((B, Hq), **f32)
    ws = torch.empty(ra.decode_shared_prefix_workspace_size(B, Hq, Hkv, mk, mp), **u8)
    lp, lp_lse = torch.empty((N,), **f32), torch.empty((N,), **f32)
    lpp, lpp_lse = torch.empty((N,), **f32), torch.empty((N,), **f32)
    ws_l = torch.empty(ra.token_logprob_workspace_size(N, V, D), **u8)
    ws_p = torch.empty(ra.token_logprob_workspace_size(N, V, D), **u8)

    def step():
        ra.decode_shared_prefix(q, kv, lens_t, gs_t, pre_t, mg, mp, mk, SCALE, out=out, lse=lse,
                                workspace=ws)
        ra.token_logprob(h, W, targets, out=lp, lse=lp_lse, workspace=ws_l)
        ra.token_logprob_packed(h, Wp, V, targets, out=lpp, lse=lpp_lse, workspace=ws_p)

    replay_and_check(step, (out, lse, lp, lp_lse, lpp, lpp_lse),
                     ("shared-prefix decode", "shared-prefix lse", "logprob N=600",
                      "logprob N=600 lse", "packed logprob N=600", "packed logprob N=600 lse"),
                     (k_pool, v_pool))
