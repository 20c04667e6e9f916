"""GPU parity of the single-launch mixed step (through the C ABI) against the fp64 CPU oracle.

The mixed call computes decode rows and append rows in one persistent launch.
Its append outputs must be bitwise those of the append call (the same tile
code, scheduled differently); its decode outputs are the decode definition
(checked against the oracle at the attention tolerance of tests.gpu_util) and
agree with the decode call up to rounding (its splits are summed by 8 waves
instead of 4).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2603_18815_amd as ra
import synth
from tests.gpu_util import APPEND_LSE_ATOL, assert_attn_close, bits, compact_rows, sample_rows

pytestmark = pytest.mark.gpu
SCALE = 1.0 / math.sqrt(128)


def i32(x, dev):
    return torch.as_tensor(np.ascontiguousarray(np.asarray(x, np.int32)), device=dev)


def say(msg):
    print(f"[gpu-test] {msg}", flush=True)


def small_mixed(seed, B, Hq, Hkv, frac=0.35):
    return synth.mixed_workload(seed, B, Hq, Hkv, frac,
                                lambda r, n: synth.uniform_int(r, n, 0, 1500),
                                lambda r, n: synth.uniform_int(r, n, 1, 300),
                                f"small mixed B={B} Hq={Hq} Hkv={Hkv}")


def caches(w, t, dev):
    return (ra.PagedKV(t.k_pool, t.v_pool, i32(w.decode_table(), dev)),
            ra.PagedKV(t.k_pool, t.v_pool, i32(w.append_table(), dev)))


def run_mixed(w, t, dev, kv_lens=None, **kw):
    kd, ka = caches(w, t, dev)
    lens = w.kv_lens if kv_lens is None else kv_lens
    return ra.mixed(t.q_decode, kd, i32(lens, dev), t.q_append, i32(w.cu_q(), dev),
                    i32(w.ctx_lens, dev), ka, int(max(lens.max(), 0)) if lens.size else 0,
                    int(w.q_lens.max()) if w.q_lens.size else 0,
                    int((w.ctx_lens + w.q_lens).max()) if w.q_lens.size else 0, SCALE,
                    want_lse=True, **kw)


@pytest.mark.parametrize("Hq,Hkv", [(32, 8), (8, 8), (16, 1), (64, 8), (32, 1)])
def test_mixed_small_vs_oracle_and_separate_calls(device, Hq, Hkv):
    w = small_mixed(Hq + Hkv, 24, Hq, Hkv)
    say(f"mixed {w.name}: {w.decode_rows.size} decode rows, {w.append_rows.size} append rows")
    t = synth.make_tensors(w, device)
    kv_lens = w.kv_lens.copy()
    kv_lens[0] = 0                        # an empty decode row: out 0, lse -inf
    od, oa, ld, la = run_mixed(w, t, device, kv_lens=kv_lens)
    kd, ka = caches(w, t, device)
    sd, sld = ra.decode(t.q_decode, kd, i32(kv_lens, device), int(kv_lens.max()), SCALE,
                        want_lse=True)
    sa, sla = ra.append(t.q_append, i32(w.cu_q(), device), i32(w.ctx_lens, device), ka,
                        int(w.q_lens.max()), int((w.ctx_lens + w.q_lens).max()), SCALE,
                        want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(oa, sa) and torch.equal(la, sla), "append part differs from append()"
    assert torch.all(od[0] == 0) and torch.all(torch.isneginf(ld[0]))
    ref_d, ref_ld = oracle.decode(bits(t.q_decode), bits(t.k_pool), bits(t.v_pool),
                                  w.decode_table(), kv_lens, SCALE)
    assert_attn_close(od.cpu().numpy()[1:], ref_d[1:], f"mixed decode G={Hq // Hkv}")
    np.testing.assert_allclose(ld.cpu().numpy()[1:], ref_ld[1:], atol=1e-4, rtol=0)
    assert_attn_close(od.cpu().numpy(), sd.cpu().numpy(), "mixed decode vs decode()")
    ref_a, ref_la = oracle.append(bits(t.q_append), w.cu_q(), w.ctx_lens, bits(t.k_pool),
                                  bits(t.v_pool), w.append_table(), SCALE)
    assert_attn_close(oa.cpu().numpy(), ref_a, f"mixed append G={Hq // Hkv}")
    np.testing.assert_allclose(la.cpu().numpy(), ref_la, atol=APPEND_LSE_ATOL, rtol=0)


def test_mixed_one_side_empty(device):
    """Only decode rows, then only append rows: the same results as the separate calls."""
    w = small_mixed(7, 16, 32, 8)
    t = synth.make_tensors(w, device)
    kd, ka = caches(w, t, device)
    e32 = torch.zeros(0, dtype=torch.int32, device=device)
    eq = t.q_append[:0]
    od, oa, _, _ = ra.mixed(t.q_decode, kd, i32(w.kv_lens, device), eq,
                            torch.zeros(1, dtype=torch.int32, device=device), e32, ka,
                            int(w.kv_lens.max()), 0, 0, SCALE)
    assert oa.shape[0] == 0
    od2, oa2, _, _ = ra.mixed(t.q_decode[:0], kd, e32, t.q_append, i32(w.cu_q(), device),
                              i32(w.ctx_lens, device), ka, 0, int(w.q_lens.max()),
                              int((w.ctx_lens + w.q_lens).max()), SCALE)
    sa, _ = ra.append(t.q_append, i32(w.cu_q(), device), i32(w.ctx_lens, device), ka,
                      int(w.q_lens.max()), int((w.ctx_lens + w.q_lens).max()), SCALE)
    torch.cuda.synchronize()
    assert od2.shape[0] == 0
    assert torch.equal(oa2, sa)
    ref_d, _ = oracle.decode(bits(t.q_decode), bits(t.k_pool), bits(t.v_pool), w.decode_table(),
                             w.kv_lens, SCALE)
    assert_attn_close(od.cpu().numpy(), ref_d, "mixed, decode rows only")


def test_mixed_poison_determinism_and_workspace_reuse(device):
    """NaN in pages no row owns is bitwise invisible; repeated calls on one workspace
    (the second over fewer rows) agree bitwise with fresh ones."""
    w = small_mixed(11, 20, 32, 8)
    t = synth.make_tensors(w, device)
    kd, ka = caches(w, t, device)
    Bd = w.kv_lens.size
    ws = torch.empty(ra.mixed_workspace_size(Bd, w.q_lens.size, 32, 8, 8, int(w.kv_lens.max()),
                                             int(w.q_lens.max())),
                     dtype=torch.uint8, device=device)
    a = run_mixed(w, t, device, workspace=ws)
    b = run_mixed(w, t, device, workspace=ws)
    # a smaller call on the same workspace: the first half of the decode rows only
    h = Bd // 2
    e32 = torch.zeros(0, dtype=torch.int32, device=device)
    small = ra.mixed(t.q_decode[:h].contiguous(), kd, i32(w.kv_lens[:h], device),
                     t.q_append[:0], torch.zeros(1, dtype=torch.int32, device=device), e32, ka,
                     int(w.kv_lens.max()), 0, 0, SCALE, workspace=ws)
    synth.poison_unowned(t.k_pool, t.v_pool, w.layout)
    c = run_mixed(w, t, device, workspace=ws)
    torch.cuda.synchronize()
    for x, y in ((a, b), (a, c)):
        for u, v in zip(x, y):
            assert torch.equal(u, v)
    assert torch.equal(small[0], a[0][:h])


def test_mixed_rollout_workload_sampled(device):
    """The 512-row step (85 % decode / 15 % append) at full size: sampled decode rows and
    sampled queries against the oracle, every append output bitwise against append()."""
    w = synth.config(5)
    say(f"mixed single launch {w.name}")
    t = synth.make_tensors(w, device)
    bt, cu, start = synth.write_plan(w)
    kv_all = ra.PagedKV(t.k_pool, t.v_pool, i32(bt, device))
    ra.kv_page_write(t.k_new, t.v_new, i32(cu, device), i32(start, device), kv_all)
    od, oa, ld, la = run_mixed(w, t, device)
    kd, ka = caches(w, t, device)
    sd, _ = ra.decode(t.q_decode, kd, i32(w.kv_lens, device), int(w.kv_lens.max()), SCALE)
    sa, _ = ra.append(t.q_append, i32(w.cu_q(), device), i32(w.ctx_lens, device), ka,
                      int(w.q_lens.max()), int((w.ctx_lens + w.q_lens).max()), SCALE)
    torch.cuda.synchronize()
    assert torch.equal(oa, sa), "append part differs from append()"
    assert_attn_close(od.cpu().numpy(), sd.cpu().numpy(), "mixed decode vs decode(), all rows")
    rows = sample_rows(w.kv_lens, 6, seed=5)
    k, v, btc = compact_rows(t.k_pool, t.v_pool, w.decode_table()[rows], w.kv_lens[rows])
    ref, ref_lse = oracle.decode(bits(t.q_decode[torch.as_tensor(rows, device=device)]), k, v,
                                 btc, w.kv_lens[rows], SCALE)
    sel = torch.as_tensor(rows, device=device)
    assert_attn_close(od[sel].cpu().numpy(), ref, "mixed decode rows vs oracle")
    np.testing.assert_allclose(ld[sel].cpu().numpy(), ref_lse, atol=1e-4, rtol=0)
    # sampled append queries: query i of row b is a one-token chunk at ctx_b + i
    rng = np.random.default_rng(55)
    arows = sample_rows(w.ctx_lens + w.q_lens, 5, seed=55)
    cuq = w.cu_q()
    sel_q, ctx1, trow = [], [], []
    for r in arows:
        T = int(w.q_lens[r])
        for i in sorted(set([0, T - 1] + rng.integers(0, T, 3).tolist())):
            sel_q.append(int(cuq[r]) + i)
            ctx1.append(int(w.ctx_lens[r]) + i)
            trow.append(r)
    table = w.append_table()[np.array(trow)]
    k, v, bt1 = compact_rows(t.k_pool, t.v_pool, table, np.array(ctx1) + 1)
    n = len(sel_q)
    ref, ref_lse = oracle.append(bits(t.q_append[torch.as_tensor(sel_q, device=device)]),
                                 np.arange(n + 1, dtype=np.int32), np.array(ctx1, np.int32),
                                 k, v, bt1, SCALE)
    qi = torch.as_tensor(sel_q, device=device)
    assert_attn_close(oa[qi].cpu().numpy(), ref, f"mixed append queries vs oracle ({n})")
    np.testing.assert_allclose(la[qi].cpu().numpy(), ref_lse, atol=APPEND_LSE_ATOL, rtol=0)
