"""GPU parity at the head counts the ABI accepts beyond the Qwen3 shapes.

Append, the fused write + append, the mixed step and decode with more than 8
KV heads (so that an XCD work queue of the planned launch holds several KV
heads: queue q takes heads q, q + 8, q + 16, ...), and append with more than 32
query heads per KV head (a tile then covers 256 / G queries, down to one).
Every expected value comes from the fp64 oracle on host copies of the same
seeded inputs; the fused and mixed calls must also equal the separate calls
bitwise where the header promises it.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2603_18815_amd as ra
import synth
from tests.gpu_util import APPEND_LSE_ATOL, assert_attn_close, bits

pytestmark = pytest.mark.gpu
SCALE = 1.0 / math.sqrt(128)
CTX = [0, 1, 15, 16, 17, 100, 300, 2000]
T = [5, 64, 1, 63, 65, 200, 130, 17]
KS, VS = 2.0 ** -5, 0.04   # fp8 pool scales


def i32(x, dev):
    return torch.as_tensor(np.ascontiguousarray(np.asarray(x, np.int32)), device=dev)


def say(msg):
    print(f"[gpu-test] {msg}", flush=True)


def pools(seed, row_tokens, Hkv, dev, fp8):
    rng = np.random.default_rng(seed)
    lay = synth.make_layout(rng, row_tokens)
    gen = synth.value_generator(seed, dev)
    if fp8:
        k = synth.randn_fp8_codes((lay.num_pages, Hkv, 16, 128), gen, dev, KS)
        v = synth.randn_fp8_codes((lay.num_pages, Hkv, 128, 16), gen, dev, VS)
    else:
        k = synth.randn_bf16((lay.num_pages, Hkv, 16, 128), gen, dev)
        v = synth.randn_bf16((lay.num_pages, Hkv, 128, 16), gen, dev)
    return lay, k, v, gen


def paged(k, v, bt, dev, fp8):
    return ra.PagedKV(k, v, i32(bt, dev), *((KS, VS) if fp8 else (None, None)))


def oracle_append(q, cu, ctx, k, v, bt, fp8):
    if fp8:
        return oracle.append_fp8(bits(q), cu, ctx, bits(k), bits(v), KS, VS, bt, SCALE)
    return oracle.append(bits(q), cu, ctx, bits(k), bits(v), bt, SCALE)


def oracle_decode(q, k, v, bt, lens, fp8):
    if fp8:
        return oracle.decode_fp8(bits(q), bits(k), bits(v), KS, VS, bt, lens, SCALE)
    return oracle.decode(bits(q), bits(k), bits(v), bt, lens, SCALE)


HEADS = [(Hkv, G) for Hkv in (12, 16, 32) for G in (1, 2, 4)]


@pytest.mark.parametrize("fp8", [False, True], ids=["bf16", "fp8"])
@pytest.mark.parametrize("Hkv,G", HEADS)
def test_append_many_kv_heads(device, Hkv, G, fp8):
    Hq = Hkv * G
    say(f"append Hkv={Hkv} G={G} fp8={fp8}")
    lay, k, v, gen = pools(1000 + Hkv * 8 + G, [c + t for c, t in zip(CTX, T)], Hkv, device, fp8)
    cu = np.concatenate([[0], np.cumsum(T)]).astype(np.int32)
    q = synth.randn_bf16((int(cu[-1]), Hq, 128), gen, device)
    kv = paged(k, v, lay.block_table, device, fp8)
    out, lse = ra.append(q, i32(cu, device), i32(CTX, device), kv, max(T),
                         max(c + t for c, t in zip(CTX, T)), SCALE, want_lse=True)
    torch.cuda.synchronize()
    ref, ref_lse = oracle_append(q, cu, CTX, k, v, lay.block_table, fp8)
    assert_attn_close(out.cpu().numpy(), ref, f"append Hkv={Hkv} G={G} fp8={fp8}")
    np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, atol=APPEND_LSE_ATOL, rtol=0)


@pytest.mark.parametrize("fp8", [False, True], ids=["bf16", "fp8"])
@pytest.mark.parametrize("Hkv,G", [(16, 2), (32, 1), (12, 4)])
def test_append_write_many_kv_heads(device, Hkv, G, fp8):
    """The fused write + append at many KV heads: bitwise the separate calls
    (outputs, lse, both pools), and the oracle on the written pools."""
    Hq = Hkv * G
    say(f"append_write Hkv={Hkv} G={G} fp8={fp8}")
    lay, k, v, gen = pools(2000 + Hkv * 8 + G, [c + t for c, t in zip(CTX, T)], Hkv, device, fp8)
    cu = np.concatenate([[0], np.cumsum(T)]).astype(np.int32)
    n = int(cu[-1])
    q = synth.randn_bf16((n, Hq, 128), gen, device)
    k_new = synth.randn_bf16((n, Hkv, 128), gen, device)
    v_new = synth.randn_bf16((n, Hkv, 128), gen, device)
    max_kv = max(c + t for c, t in zip(CTX, T))
    k1, v1, k2, v2 = k.clone(), v.clone(), k.clone(), v.clone()
    kv1 = paged(k1, v1, lay.block_table, device, fp8)
    kv2 = paged(k2, v2, lay.block_table, device, fp8)
    cu_t, ctx_t = i32(cu, device), i32(CTX, device)
    o1, l1 = ra.append_write(q, k_new, v_new, cu_t, ctx_t, kv1, max(T), max_kv, SCALE,
                             want_lse=True)
    ra.kv_page_write(k_new, v_new, cu_t, ctx_t, kv2, max(T), max_kv)
    o2, l2 = ra.append(q, cu_t, ctx_t, kv2, max(T), max_kv, SCALE, want_lse=True)
    torch.cuda.synchronize()
    for a, b in zip((o1, l1, k1, v1), (o2, l2, k2, v2)):
        assert torch.equal(a, b)
    if fp8:
        kx, vx = oracle.page_write_fp8(bits(k_new), bits(v_new), cu, CTX, lay.block_table,
                                       bits(k), bits(v), KS, VS)
    else:
        kx, vx = oracle.page_write(bits(k_new), bits(v_new), cu, CTX, lay.block_table,
                                   bits(k), bits(v))
    assert np.array_equal(bits(k1), kx) and np.array_equal(bits(v1), vx)
    ref, ref_lse = oracle_append(q, cu, CTX, k1, v1, lay.block_table, fp8)
    assert_attn_close(o1.cpu().numpy(), ref, f"append_write Hkv={Hkv} G={G} fp8={fp8}")
    np.testing.assert_allclose(l1.cpu().numpy(), ref_lse, atol=APPEND_LSE_ATOL, rtol=0)


@pytest.mark.parametrize("fp8", [False, True], ids=["bf16", "fp8"])
@pytest.mark.parametrize("Hkv,G", [(16, 1), (16, 4), (32, 2), (12, 2)])
def test_mixed_many_kv_heads(device, Hkv, G, fp8):
    """Decode rows and append rows in one launch at many KV heads: append part
    bitwise append(), both parts against the oracle."""
    Hq = Hkv * G
    w = synth.mixed_workload(3000 + Hkv * 8 + G, 20, Hq, Hkv, 0.35,
                             lambda r, n: synth.uniform_int(r, n, 0, 1200),
                             lambda r, n: synth.uniform_int(r, n, 1, 200),
                             f"mixed Hkv={Hkv} G={G}")
    say(f"{w.name} fp8={fp8}: {w.decode_rows.size} decode rows, {w.append_rows.size} append rows")
    gen = synth.value_generator(3000 + Hkv, device)
    n = w.layout.num_pages
    if fp8:
        k = synth.randn_fp8_codes((n, Hkv, 16, 128), gen, device, KS)
        v = synth.randn_fp8_codes((n, Hkv, 128, 16), gen, device, VS)
    else:
        k = synth.randn_bf16((n, Hkv, 16, 128), gen, device)
        v = synth.randn_bf16((n, Hkv, 128, 16), gen, device)
    qd = synth.randn_bf16((w.kv_lens.size, Hq, 128), gen, device)
    qa = synth.randn_bf16((int(w.q_lens.sum()), Hq, 128), gen, device)
    kd = paged(k, v, w.decode_table(), device, fp8)
    ka = paged(k, v, w.append_table(), device, fp8)
    mq, mka = int(w.q_lens.max()), int((w.ctx_lens + w.q_lens).max())
    cu_t, ctx_t = i32(w.cu_q(), device), i32(w.ctx_lens, device)
    od, oa, ld, la = ra.mixed(qd, kd, i32(w.kv_lens, device), qa, cu_t, ctx_t, ka,
                              int(w.kv_lens.max()), mq, mka, SCALE, want_lse=True)
    sa, sla = ra.append(qa, cu_t, ctx_t, ka, mq, mka, SCALE, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(oa, sa) and torch.equal(la, sla), "append part differs from append()"
    ref_d, ref_ld = oracle_decode(qd, k, v, w.decode_table(), w.kv_lens, fp8)
    assert_attn_close(od.cpu().numpy(), ref_d, f"{w.name} decode rows fp8={fp8}")
    np.testing.assert_allclose(ld.cpu().numpy(), ref_ld, atol=1e-4, rtol=0)
    ref_a, ref_la = oracle_append(qa, w.cu_q(), w.ctx_lens, k, v, w.append_table(), fp8)
    assert_attn_close(oa.cpu().numpy(), ref_a, f"{w.name} append rows fp8={fp8}")
    np.testing.assert_allclose(la.cpu().numpy(), ref_la, atol=APPEND_LSE_ATOL, rtol=0)


@pytest.mark.parametrize("fp8", [False, True], ids=["bf16", "fp8"])
@pytest.mark.parametrize("Hkv,G", [(16, 1), (16, 4), (32, 1), (32, 2), (12, 3)])
def test_decode_many_kv_heads(device, Hkv, G, fp8):
    Hq = Hkv * G
    lens = [1, 15, 16, 17, 129, 700, 2100]
    say(f"decode Hkv={Hkv} G={G} fp8={fp8}")
    lay, k, v, gen = pools(4000 + Hkv * 8 + G, lens, Hkv, device, fp8)
    q = synth.randn_bf16((len(lens), Hq, 128), gen, device)
    kv = paged(k, v, lay.block_table, device, fp8)
    out, lse = ra.decode(q, kv, i32(lens, device), max(lens), SCALE, want_lse=True)
    torch.cuda.synchronize()
    ref, ref_lse = oracle_decode(q, k, v, lay.block_table, lens, fp8)
    assert_attn_close(out.cpu().numpy(), ref, f"decode Hkv={Hkv} G={G} fp8={fp8}")
    np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, atol=1e-4, rtol=0)


@pytest.mark.parametrize("Hkv,G,fp8", [(1, 64, False), (2, 64, False), (1, 128, False),
                                       (1, 256, False), (1, 256, True), (2, 128, True)])
def test_append_large_groups(device, Hkv, G, fp8):
    """G > 32 query heads per KV head: a tile holds 256 / G queries (4, 2, 1),
    each of its waves a slice of one query's heads."""
    Hq = Hkv * G
    ctx = [0, 1, 15, 17, 300, 1000]
    t = [5, 3, 1, 9, 40, 17]
    say(f"append large group Hkv={Hkv} G={G} fp8={fp8}")
    lay, k, v, gen = pools(5000 + Hkv * 8 + G, [c + n for c, n in zip(ctx, t)], Hkv, device, fp8)
    cu = np.concatenate([[0], np.cumsum(t)]).astype(np.int32)
    q = synth.randn_bf16((int(cu[-1]), Hq, 128), gen, device)
    kv = paged(k, v, lay.block_table, device, fp8)
    out, lse = ra.append(q, i32(cu, device), i32(ctx, device), kv, max(t),
                         max(c + n for c, n in zip(ctx, t)), SCALE, want_lse=True)
    torch.cuda.synchronize()
    ref, ref_lse = oracle_append(q, cu, ctx, k, v, lay.block_table, fp8)
    assert_attn_close(out.cpu().numpy(), ref, f"append Hkv={Hkv} G={G} fp8={fp8}")
    np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, atol=APPEND_LSE_ATOL, rtol=0)
