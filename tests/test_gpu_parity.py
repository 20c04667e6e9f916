"""GPU parity of the HIP library (through the C ABI) against the fp64 CPU oracle.

Every expected value comes from `oracle/` on host copies of the same seeded
inputs (or, for bitwise invariants, from a second run of the library on
rearranged inputs). Floating-point outputs must satisfy max-abs <= 1e-2 and
rel-L2 <= 5e-3 over each compared tensor; page writes and gathers must be
bit-exact over the whole pool.
"""
import math
import os

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


def small_pool(seed, row_tokens, Hkv, dev, extra_stride=0):
    rng = np.random.default_rng(seed)
    lay = synth.make_layout(rng, row_tokens, extra_stride=extra_stride)
    gen = synth.value_generator(seed, dev)
    k = synth.randn_bf16((lay.num_pages, Hkv, 16, 128), gen, dev)
    v = synth.randn_bf16((lay.num_pages, Hkv, 128, 16), gen, dev)
    return lay, k, v, gen


# ------------------------------------------------------------------ page write / gather

def test_page_write_bitexact_ragged(device):
    say("page_write ragged")
    starts = [0, 5, 16, 15, 33, 0, 100, 31]
    news = [1, 20, 16, 2, 40, 0, 7, 33]
    lay, k, v, gen = small_pool(11, [s + n + 3 for s, n in zip(starts, news)], 2, device)
    cu = np.concatenate([[0], np.cumsum(news)]).astype(np.int32)
    k_new = synth.randn_bf16((int(cu[-1]), 2, 128), gen, device)
    v_new = synth.randn_bf16((int(cu[-1]), 2, 128), gen, device)
    kh, vh = bits(k), bits(v)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device))
    ra.kv_page_write(k_new, v_new, i32(cu, device), i32(starts, device), kv)
    torch.cuda.synchronize()
    kx, vx = oracle.page_write(bits(k_new), bits(v_new), cu, starts, lay.block_table, kh, vh)
    np.testing.assert_array_equal(bits(k), kx)
    np.testing.assert_array_equal(bits(v), vx)


def test_page_write_bitexact_append_workload(device):
    """The full page-write plan of the append workload (33.8k tokens), whole pool compared."""
    w = synth.config(3)
    say(f"page_write {w.name}")
    t = synth.make_tensors(w, device)
    bt, cu, start = synth.write_plan(w)
    kh, vh = bits(t.k_pool), bits(t.v_pool)
    kv = ra.PagedKV(t.k_pool, t.v_pool, i32(bt, device))
    ra.kv_page_write(t.k_new, t.v_new, i32(cu, device), i32(start, device), kv)
    torch.cuda.synchronize()
    kx, vx = oracle.page_write(bits(t.k_new), bits(t.v_new), cu, start, bt, kh, vh)
    np.testing.assert_array_equal(bits(t.k_pool), kx)
    np.testing.assert_array_equal(bits(t.v_pool), vx)


@pytest.mark.parametrize("case", ["config1", "ragged"])
def test_page_gather_bitexact(device, case):
    say(f"page_gather {case}")
    if case == "config1":
        w = synth.config(1)
        t = synth.make_tensors(w, device)
        lay, k, v = w.layout, t.k_pool, t.v_pool
        Hkv = w.Hkv
    else:
        Hkv = 3
        lay, k, v, _ = small_pool(5, [1, 16, 17, 40, 0, 33], Hkv, device)
    lens = lay.row_tokens
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device))
    ko, vo = ra.kv_page_gather(kv, i32(lens, device), i32(cu, device))
    torch.cuda.synchronize()
    kx, vx = oracle.page_gather(bits(k), bits(v), lay.block_table, lens, cu)
    np.testing.assert_array_equal(bits(ko), kx)
    np.testing.assert_array_equal(bits(vo), vx)


# ----------------------------------------------------------------------------- decode

def run_decode(w, t, dev, rows=None, **kw):
    kv = ra.PagedKV(t.k_pool, t.v_pool, i32(w.decode_table(), dev))
    return ra.decode(t.q_decode, kv, i32(w.kv_lens, dev), int(w.kv_lens.max()), SCALE,
                     want_lse=True, **kw)


def test_decode_parity_small_workload_full(device):
    w = synth.config(1)
    say(f"decode {w.name}")
    t = synth.make_tensors(w, device)
    out, lse = run_decode(w, t, device)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.decode(bits(t.q_decode), bits(t.k_pool), bits(t.v_pool),
                                 w.decode_table(), w.kv_lens, SCALE)
    assert_attn_close(out.cpu().numpy(), ref, "decode config 1")
    np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, atol=1e-4, rtol=0)


@pytest.mark.parametrize("c", [2, 4])
def test_decode_parity_full_size_sampled_rows(device, c):
    w = synth.config(c)
    say(f"decode {w.name}")
    t = synth.make_tensors(w, device)
    out, lse = run_decode(w, t, device)
    torch.cuda.synchronize()
    rows = sample_rows(w.kv_lens, 8, seed=c)
    k, v, bt = compact_rows(t.k_pool, t.v_pool, w.decode_table()[rows], w.kv_lens[rows])
    ref, ref_lse = oracle.decode(bits(t.q_decode[torch.as_tensor(rows, device=device)]), k, v,
                                 bt, w.kv_lens[rows], SCALE)
    assert_attn_close(out[torch.as_tensor(rows, device=device)].cpu().numpy(), ref,
                      f"decode config {c} rows {rows.tolist()}")
    np.testing.assert_allclose(lse[torch.as_tensor(rows, device=device)].cpu().numpy(), ref_lse,
                               atol=1e-4, rtol=0)


@pytest.mark.parametrize("Hq,Hkv", [(8, 8), (4, 2), (32, 8), (64, 8), (32, 2), (24, 1), (32, 1)])
def test_decode_edge_lengths_and_groups(device, Hq, Hkv):
    lens = [1, 2, 15, 16, 17, 31, 32, 33, 127, 128, 129, 300, 1000]
    say(f"decode edges Hq={Hq} Hkv={Hkv}")
    lay, k, v, gen = small_pool(Hq + Hkv, lens, Hkv, device, extra_stride=2)
    q = synth.randn_bf16((len(lens), Hq, 128), gen, device)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device))
    out, lse = ra.decode(q, kv, i32(lens, device), max(lens), SCALE, want_lse=True)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.decode(bits(q), bits(k), bits(v), lay.block_table, lens, SCALE)
    assert_attn_close(out.cpu().numpy(), ref, f"decode edges G={Hq // Hkv}")
    np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, atol=1e-4, rtol=0)
    # one cached key: the output is that value row, exactly
    G = Hq // Hkv
    vrow = v[int(lay.block_table[0, 0])][:, :, 0].float().cpu()          # [Hkv][128]
    np.testing.assert_array_equal(out[0].cpu().numpy(),
                                  vrow.repeat_interleave(G, 0).numpy())


def test_decode_empty_rows(device):
    lens = [0, 5, 0]
    lay, k, v, gen = small_pool(3, [1, 5, 1], 2, device)
    q = synth.randn_bf16((3, 4, 128), gen, device)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device))
    out, lse = ra.decode(q, kv, i32(lens, device), 5, SCALE, want_lse=True)
    torch.cuda.synchronize()
    assert torch.all(out[0] == 0) and torch.all(out[2] == 0)
    assert torch.all(torch.isneginf(lse[0])) and torch.all(torch.isneginf(lse[2]))
    assert torch.all(torch.isfinite(out[1]))


def test_decode_poison_is_bitwise_invisible(device):
    w = synth.config(1)
    t = synth.make_tensors(w, device)
    clean, clean_lse = run_decode(w, t, device)
    synth.poison_unowned(t.k_pool, t.v_pool, w.layout)
    dirty, dirty_lse = run_decode(w, t, device)
    torch.cuda.synchronize()
    assert torch.equal(clean, dirty) and torch.equal(clean_lse, dirty_lse)


def _scatter_rows(K, V, lay, Hkv, dev, fill_nan=False):
    """Place dense rows K/V ([R][Hkv][L][128] lists) on pages with torch indexing."""
    k = torch.empty((lay.num_pages, Hkv, 16, 128), dtype=torch.bfloat16, device=dev)
    v = torch.empty((lay.num_pages, Hkv, 128, 16), dtype=torch.bfloat16, device=dev)
    k.fill_(float("nan") if fill_nan else 0.0)
    v.fill_(float("nan") if fill_nan else 0.0)
    for r, (kr, vr) in enumerate(zip(K, V)):
        L = kr.shape[1]
        j = torch.arange(L, device=dev)
        pg = torch.as_tensor(lay.block_table[r], device=dev).long()[j // 16]
        k[pg, :, j % 16, :] = kr.transpose(0, 1)
        v[pg, :, :, j % 16] = vr.transpose(0, 1)
    return k, v


def test_decode_page_permutation_is_bitwise_invisible(device):
    lens = [700, 33, 2048, 1]
    Hkv, Hq = 2, 8
    gen = synth.value_generator(77, device)
    K = [synth.randn_bf16((Hkv, L, 128), gen, device) for L in lens]
    V = [synth.randn_bf16((Hkv, L, 128), gen, device) for L in lens]
    q = synth.randn_bf16((len(lens), Hq, 128), gen, device)
    outs = []
    for seed in (1, 2):
        lay = synth.make_layout(np.random.default_rng(seed), lens)
        k, v = _scatter_rows(K, V, lay, Hkv, device)
        kv = ra.PagedKV(k, v, i32(lay.block_table, device))
        outs.append(ra.decode(q, kv, i32(lens, device), max(lens), SCALE, want_lse=True))
    torch.cuda.synchronize()
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


def test_decode_deterministic_and_split_invariant(device):
    w = synth.config(2)
    t = synth.make_tensors(w, device)
    a, la = run_decode(w, t, device)
    b, lb = run_decode(w, t, device)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(la, lb)
    os.environ["RA_SPLIT_TOKENS"] = "128"
    try:
        c, lc = run_decode(w, t, device)
        torch.cuda.synchronize()
    finally:
        del os.environ["RA_SPLIT_TOKENS"]
    rel = (torch.linalg.vector_norm(a - c) / torch.linalg.vector_norm(a)).item()
    say(f"split invariance rel={rel:.3e}")
    assert rel < 1e-5
    assert (la - lc).abs().max().item() < 1e-4


# ----------------------------------------------------------------------------- append

def run_append(w, t, dev, q=None):
    kv = ra.PagedKV(t.k_pool, t.v_pool, i32(w.append_table(), dev))
    return ra.append(t.q_append if q is None else q, i32(w.cu_q(), dev), i32(w.ctx_lens, dev),
                     kv, int(w.q_lens.max()), int((w.ctx_lens + w.q_lens).max()), SCALE,
                     want_lse=True)


def _append_small(dev, seed, ctx, T, Hq, Hkv):
    lens = [c + n for c, n in zip(ctx, T)]
    lay, k, v, gen = small_pool(seed, lens, Hkv, dev)
    cu = np.concatenate([[0], np.cumsum(T)]).astype(np.int32)
    q = synth.randn_bf16((int(cu[-1]), Hq, 128), gen, dev)
    return lay, k, v, q, cu


@pytest.mark.parametrize("Hq,Hkv", [(32, 8), (8, 8), (64, 8), (6, 2), (16, 1)])
def test_append_parity_ragged(device, Hq, Hkv):
    ctx = [0, 1, 15, 16, 17, 100, 300, 2000]
    T = [5, 64, 1, 63, 65, 200, 130, 17]
    say(f"append ragged Hq={Hq} Hkv={Hkv}")
    lay, k, v, q, cu = _append_small(device, Hq * 7 + Hkv, ctx, T, Hq, Hkv)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device))
    out, lse = ra.append(q, i32(cu, device), i32(ctx, device), kv, max(T),
                         max(c + n for c, n in zip(ctx, T)), SCALE, want_lse=True)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.append(bits(q), cu, ctx, bits(k), bits(v), lay.block_table, SCALE)
    assert_attn_close(out.cpu().numpy(), ref, f"append ragged G={Hq // Hkv}")
    np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, atol=APPEND_LSE_ATOL, rtol=0)


def _oracle_sampled_queries(w, t, rows, per_row, seed, dev):
    """Oracle on sampled queries: query i of row b equals a one-token chunk at ctx_b + i."""
    rng = np.random.default_rng(seed)
    cu = w.cu_q()
    sel_rows, sel_q, ctx1 = [], [], []
    for r in rows:
        T = int(w.q_lens[r])
        qs = sorted(set([0, T - 1] + rng.integers(0, T, per_row).tolist()))
        for i in qs:
            sel_rows.append(r)
            sel_q.append(int(cu[r]) + i)
            ctx1.append(int(w.ctx_lens[r]) + i)
    table = w.append_table()[np.array(sel_rows)]
    k, v, bt = compact_rows(t.k_pool, t.v_pool, table, np.array(ctx1) + 1)
    qsel = bits(t.q_append[torch.as_tensor(sel_q, device=dev)])
    n = len(sel_q)
    ref, ref_lse = oracle.append(qsel, np.arange(n + 1, dtype=np.int32), np.array(ctx1, np.int32),
                                 k, v, bt, SCALE)
    return np.array(sel_q), ref, ref_lse


@pytest.mark.parametrize("c", [3])
def test_append_parity_full_size_sampled(device, c):
    w = synth.config(c)
    say(f"append {w.name}")
    t = synth.make_tensors(w, device)
    out, lse = run_append(w, t, device)
    torch.cuda.synchronize()
    rows = sample_rows(w.ctx_lens + w.q_lens, 8, seed=c)
    sel, ref, ref_lse = _oracle_sampled_queries(w, t, rows, 6, c, device)
    idx = torch.as_tensor(sel, device=device)
    assert_attn_close(out[idx].cpu().numpy(), ref, f"append config {c} ({len(sel)} queries)")
    np.testing.assert_allclose(lse[idx].cpu().numpy(), ref_lse, atol=APPEND_LSE_ATOL, rtol=0)


def test_append_one_token_matches_decode(device):
    ctx = [0, 15, 16, 500, 4095]
    T = [1] * 5
    lay, k, v, q, cu = _append_small(device, 99, ctx, T, 32, 8)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device))
    oa, la = ra.append(q, i32(cu, device), i32(ctx, device), kv, 1, max(ctx) + 1, SCALE,
                       want_lse=True)
    od, ld = ra.decode(q, kv, i32([c + 1 for c in ctx], device), max(ctx) + 1, SCALE,
                       want_lse=True)
    torch.cuda.synchronize()
    ref, _ = oracle.decode(bits(q), bits(k), bits(v), lay.block_table, [c + 1 for c in ctx],
                           SCALE)
    assert_attn_close(oa.cpu().numpy(), ref, "append T=1")
    assert_attn_close(od.cpu().numpy(), ref, "decode L=ctx+1")
    assert_attn_close(oa.cpu().numpy(), od.cpu().numpy(), "append T=1 vs decode")


def test_append_causal_future_keys_are_bitwise_invisible(device):
    ctx, T = [300, 40], [200, 90]
    lay, k, v, q, cu = _append_small(device, 123, ctx, T, 32, 8)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device))
    args = (i32(cu, device), i32(ctx, device), kv, max(T), 500, SCALE)
    base, base_lse = ra.append(q, *args, want_lse=True)
    cut = 57                                  # query index inside row 0
    gen = synth.value_generator(5, device)
    for j in range(ctx[0] + cut + 1, ctx[0] + T[0]):     # rewrite every later key of row 0
        pg = int(lay.block_table[0, j // 16])
        k[pg, :, j % 16, :] = synth.randn_bf16((8, 128), gen, device)
        v[pg, :, :, j % 16] = synth.randn_bf16((8, 128), gen, device)
    new, new_lse = ra.append(q, *args, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(new[:cut + 1], base[:cut + 1])
    assert torch.equal(new_lse[:cut + 1], base_lse[:cut + 1])
    assert not torch.equal(new[cut + 1:T[0]], base[cut + 1:T[0]])
    assert torch.equal(new[T[0]:], base[T[0]:])          # the other row is untouched


def test_append_poison_and_determinism(device):
    ctx, T = [0, 17, 250, 1000], [33, 100, 64, 7]
    lay, k, v, q, cu = _append_small(device, 321, ctx, T, 32, 8)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device))
    args = (i32(cu, device), i32(ctx, device), kv, max(T), 1007, SCALE)
    a, la = ra.append(q, *args, want_lse=True)
    b, lb = ra.append(q, *args, want_lse=True)
    synth.poison_unowned(k, v, lay)
    c, lc = ra.append(q, *args, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(la, lb)
    assert torch.equal(a, c) and torch.equal(la, lc)


# --------------------------------------------------------------------- mixed rollout step

def test_mixed_rollout_step_sampled(device):
    """Page write of the step's new tokens, then decode rows and append rows on one pool."""
    w = synth.config(5)
    say(f"mixed {w.name}")
    t = synth.make_tensors(w, device)
    bt, cu, start = synth.write_plan(w)
    kv_all = ra.PagedKV(t.k_pool, t.v_pool, i32(bt, device))
    ra.kv_page_write(t.k_new, t.v_new, i32(cu, device), i32(start, device), kv_all)
    dec, dec_lse = run_decode(w, t, device)
    app, app_lse = run_append(w, t, device)
    torch.cuda.synchronize()
    # the step's written tokens are in place (gather of the new positions, bit-exact)
    nd = w.decode_rows.size
    new_tok = bits(t.k_new)
    rows = sample_rows(w.kv_lens, 6, seed=5)
    k, v, btc = compact_rows(t.k_pool, t.v_pool, w.decode_table()[rows], w.kv_lens[rows])
    for i, r in enumerate(rows):
        pos = int(w.kv_lens[r]) - 1
        pg = btc[i, pos // 16]
        np.testing.assert_array_equal(k[pg, :, pos % 16, :], new_tok[r])
    ref, _ = oracle.decode(bits(t.q_decode[torch.as_tensor(rows, device=device)]), k, v, btc,
                           w.kv_lens[rows], SCALE)
    assert_attn_close(dec[torch.as_tensor(rows, device=device)].cpu().numpy(), ref,
                      "mixed decode rows")
    arows = sample_rows(w.ctx_lens + w.q_lens, 6, seed=55)
    sel, ref, _ = _oracle_sampled_queries(w, t, arows, 4, 5, device)
    assert_attn_close(app[torch.as_tensor(sel, device=device)].cpu().numpy(), ref,
                      f"mixed append rows ({len(sel)} queries)")
    assert nd + w.append_rows.size == 512
