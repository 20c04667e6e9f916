"""GPU checks of the fused page write + append (rollout_attn_append_write).

The fused call must equal, bitwise, kv_page_write followed by append on the
same inputs: the outputs, the lse and both whole pools. The attention itself
is also compared with the fp64 oracle (tolerance of tests.gpu_util).
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


def i32(x, dev):
    return torch.as_tensor(np.ascontiguousarray(np.asarray(x, np.int32)), device=dev)


def say(msg):
    print(f"[gpu-test] {msg}", flush=True)


def two_ways(q, k_new, v_new, cu, ctx, k, v, bt, max_q, max_kv, dev, scales=None):
    """(fused result, separate result), each on its own copy of the pools
    (fp8 pools when scales = (k_scale, v_scale))."""
    k1, v1, k2, v2 = k.clone(), v.clone(), k.clone(), v.clone()
    sc = scales or (None, None)
    kv1 = ra.PagedKV(k1, v1, i32(bt, dev), *sc)
    kv2 = ra.PagedKV(k2, v2, i32(bt, dev), *sc)
    cu_t, ctx_t = i32(cu, dev), i32(ctx, dev)
    o1, l1 = ra.append_write(q, k_new, v_new, cu_t, ctx_t, kv1, max_q, max_kv, SCALE,
                             want_lse=True)
    ra.kv_page_write(k_new, v_new, cu_t, ctx_t, kv2, max_q, max_kv)
    o2, l2 = ra.append(q, cu_t, ctx_t, kv2, max_q, max_kv, SCALE, want_lse=True)
    torch.cuda.synchronize()
    return (o1, l1, k1, v1), (o2, l2, k2, v2)


@pytest.mark.parametrize("Hq,Hkv", [(32, 8), (8, 8), (16, 1), (6, 2)])
def test_append_write_equals_write_then_append(device, Hq, Hkv):
    ctx = [0, 1, 15, 16, 17, 100, 300, 2000]
    T = [5, 64, 1, 63, 65, 200, 130, 17]
    say(f"append_write Hq={Hq} Hkv={Hkv}")
    rng = np.random.default_rng(Hq + Hkv)
    lay = synth.make_layout(rng, [c + t for c, t in zip(ctx, T)])
    gen = synth.value_generator(Hq * 3 + Hkv, device)
    k = synth.randn_bf16((lay.num_pages, Hkv, 16, 128), gen, device)
    v = synth.randn_bf16((lay.num_pages, Hkv, 128, 16), gen, device)
    cu = np.concatenate([[0], np.cumsum(T)]).astype(np.int32)
    n = int(cu[-1])
    q = synth.randn_bf16((n, Hq, 128), gen, device)
    k_new = synth.randn_bf16((n, Hkv, 128), gen, device)
    v_new = synth.randn_bf16((n, Hkv, 128), gen, device)
    # the slots the chunks will occupy hold NaN before the call: nothing may read them
    for b in range(len(ctx)):
        for pos in range(ctx[b], ctx[b] + T[b]):
            pg = int(lay.block_table[b, pos // 16])
            k[pg, :, pos % 16, :] = float("nan")
            v[pg, :, :, pos % 16] = float("nan")
    max_kv = max(c + t for c, t in zip(ctx, T))
    f, s = two_ways(q, k_new, v_new, cu, ctx, k, v, lay.block_table, max(T), max_kv, device)
    for a, b in zip(f, s):
        assert torch.equal(a, b)
    ref, ref_lse = oracle.append(bits(q), cu, ctx, bits(s[2]), bits(s[3]), lay.block_table,
                                 SCALE)
    assert_attn_close(f[0].cpu().numpy(), ref, f"append_write G={Hq // Hkv}")
    np.testing.assert_allclose(f[1].cpu().numpy(), ref_lse, atol=APPEND_LSE_ATOL, rtol=0)


def test_append_write_full_append_workload(device):
    """The B=32 append workload: fused vs separate, bitwise (outputs, lse, pools)."""
    w = synth.config(3)
    say(f"append_write {w.name}")
    t = synth.make_tensors(w, device)
    bt = w.append_table()
    cu, ctx = w.cu_q(), w.ctx_lens
    n = int(cu[-1])
    k_new, v_new = t.k_new[-n:].contiguous(), t.v_new[-n:].contiguous()
    f, s = two_ways(t.q_append, k_new, v_new, cu, ctx, t.k_pool, t.v_pool, bt,
                    int(w.q_lens.max()), int((w.ctx_lens + w.q_lens).max()), device)
    for a, b in zip(f, s):
        assert torch.equal(a, b)


@pytest.mark.parametrize("Hq,Hkv", [(32, 8), (16, 1)])
def test_append_write_fp8_equals_write_then_append(device, Hq, Hkv):
    """fp8 pools: the fused call quantizes the chunk exactly as kv_page_write does
    (whole pools bitwise) and attends the stored codes (outputs bitwise, and
    against the oracle on the written pools)."""
    ctx = [0, 1, 15, 16, 17, 100, 300, 2000]
    T = [5, 64, 1, 63, 65, 200, 130, 17]
    ks, vs = 0.04, 0.03
    say(f"append_write fp8 Hq={Hq} Hkv={Hkv}")
    rng = np.random.default_rng(Hq + Hkv + 7)
    lay = synth.make_layout(rng, [c + t for c, t in zip(ctx, T)])
    gen = synth.value_generator(Hq * 5 + Hkv, device)
    k = synth.randn_fp8_codes((lay.num_pages, Hkv, 16, 128), gen, device, ks)
    v = synth.randn_fp8_codes((lay.num_pages, Hkv, 128, 16), gen, device, vs)
    cu = np.concatenate([[0], np.cumsum(T)]).astype(np.int32)
    n = int(cu[-1])
    q = synth.randn_bf16((n, Hq, 128), gen, device)
    k_new = synth.randn_bf16((n, Hkv, 128), gen, device)
    v_new = synth.randn_bf16((n, Hkv, 128), gen, device)
    # the slots the chunks will occupy hold the NaN code before the call
    for b in range(len(ctx)):
        for pos in range(ctx[b], ctx[b] + T[b]):
            pg = int(lay.block_table[b, pos // 16])
            k[pg, :, pos % 16, :] = 0x7F
            v[pg, :, :, pos % 16] = 0x7F
    max_kv = max(c + t for c, t in zip(ctx, T))
    f, s = two_ways(q, k_new, v_new, cu, ctx, k, v, lay.block_table, max(T), max_kv, device,
                    scales=(ks, vs))
    for a, b in zip(f, s):
        assert torch.equal(a, b)
    kx, vx = oracle.page_write_fp8(bits(k_new), bits(v_new), cu, ctx, lay.block_table,
                                   bits(k), bits(v), ks, vs)
    assert np.array_equal(bits(f[2]), kx) and np.array_equal(bits(f[3]), vx)
    ref, ref_lse = oracle.append_fp8(bits(q), cu, ctx, kx, vx, ks, vs, lay.block_table, SCALE)
    assert_attn_close(f[0].cpu().numpy(), ref, f"append_write fp8 G={Hq // Hkv}")
    np.testing.assert_allclose(f[1].cpu().numpy(), ref_lse, atol=APPEND_LSE_ATOL, rtol=0)
