"""GPU checks of rotary position embedding on write (through the C ABI).

kv_page_write_rope must leave the pools bit for bit as the oracle's rotation
(oracle.rope) followed by the oracle's page write; the rounding of each
rotated element to bf16 is taken in the precision the library states for it
(fp32 products and sums), which the oracle follows, so the comparison is
exact. rollout_attn_append_write_rope must equal, bitwise, the rotated write
followed by append on the oracle-rotated queries, and meet the fp64 oracle
attention on those inputs (tolerance of tests.gpu_util).
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


def rope_table(theta, rows):
    """cos | sin of p * theta^(-2i/128) for p < rows (fp64 math, stored fp32)."""
    inv = float(theta) ** (-2.0 * np.arange(64) / 128.0)
    ang = np.arange(rows, dtype=np.float64)[:, None] * inv[None, :]
    return np.concatenate([np.cos(ang), np.sin(ang)], axis=1).astype(np.float32)


def from_bits(b, dev):
    return torch.from_numpy(np.ascontiguousarray(b).view(np.int16)).view(torch.bfloat16).to(dev)


@pytest.mark.parametrize("fp8", [False, True])
def test_page_write_rope_bitexact(device, fp8):
    """Ragged rows written at positions up to ~30k: both whole pools equal the
    oracle's rotate-then-write, bit for bit."""
    start = [0, 15, 16, 4095, 30001, 777]
    n = [1, 40, 17, 200, 33, 64]
    Hkv = 4
    say(f"kv_page_write_rope fp8={fp8}")
    rng = np.random.default_rng(31)
    lay = synth.make_layout(rng, [s + t for s, t in zip(start, n)])
    gen = synth.value_generator(31, device)
    ks, vs = 0.03, 0.02
    if fp8:
        k = synth.randn_fp8_codes((lay.num_pages, Hkv, 16, 128), gen, device, ks)
        v = synth.randn_fp8_codes((lay.num_pages, Hkv, 128, 16), gen, device, vs)
    else:
        k = synth.randn_bf16((lay.num_pages, Hkv, 16, 128), gen, device)
        v = synth.randn_bf16((lay.num_pages, Hkv, 128, 16), gen, device)
    cu = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    k_new = synth.randn_bf16((int(cu[-1]), Hkv, 128), gen, device)
    v_new = synth.randn_bf16((int(cu[-1]), Hkv, 128), gen, device)
    max_pos = max(s + t for s, t in zip(start, n))
    table = rope_table(1e6, max_pos)
    k0, v0 = bits(k), bits(v)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device), *((ks, vs) if fp8 else (None, None)))
    ra.kv_page_write(k_new, v_new, i32(cu, device), i32(start, device), kv, max(n), max_pos,
                     cos_sin=torch.from_numpy(table).to(device))
    torch.cuda.synchronize()
    pos = np.concatenate([np.arange(s, s + t) for s, t in zip(start, n)]).astype(np.int32)
    k_rot = oracle.rope(bits(k_new), pos, table)
    if fp8:
        kx, vx = oracle.page_write_fp8(k_rot, bits(v_new), cu, start, lay.block_table, k0, v0,
                                       ks, vs)
    else:
        kx, vx = oracle.page_write(k_rot, bits(v_new), cu, start, lay.block_table, k0, v0)
    assert np.array_equal(bits(k), kx), "K pool differs from the oracle's rotated write"
    assert np.array_equal(bits(v), vx), "V pool differs from the oracle's write"


@pytest.mark.parametrize("Hq,Hkv,fp8", [(32, 8, False), (16, 1, False), (32, 8, True)])
def test_append_write_rope(device, Hq, Hkv, fp8):
    ctx = [0, 1, 15, 16, 17, 100, 300, 2000]
    T = [5, 64, 1, 63, 65, 200, 130, 17]
    say(f"append_write_rope Hq={Hq} Hkv={Hkv} fp8={fp8}")
    rng = np.random.default_rng(Hq + Hkv + 32)
    lay = synth.make_layout(rng, [c + t for c, t in zip(ctx, T)])
    gen = synth.value_generator(Hq + 33, device)
    ks, vs = 0.04, 0.03
    if fp8:
        k = synth.randn_fp8_codes((lay.num_pages, Hkv, 16, 128), gen, device, ks)
        v = synth.randn_fp8_codes((lay.num_pages, Hkv, 128, 16), gen, device, vs)
    else:
        k = synth.randn_bf16((lay.num_pages, Hkv, 16, 128), gen, device)
        v = synth.randn_bf16((lay.num_pages, Hkv, 128, 16), gen, device)
    cu = np.concatenate([[0], np.cumsum(T)]).astype(np.int32)
    n = int(cu[-1])
    q = synth.randn_bf16((n, Hq, 128), gen, device)
    k_new = synth.randn_bf16((n, Hkv, 128), gen, device)
    v_new = synth.randn_bf16((n, Hkv, 128), gen, device)
    max_kv = max(c + t for c, t in zip(ctx, T))
    table = rope_table(1e6, max_kv + 5)
    tab = torch.from_numpy(table).to(device)
    sc = (ks, vs) if fp8 else (None, None)
    cu_t, ctx_t = i32(cu, device), i32(ctx, device)
    # fused
    k1, v1 = k.clone(), v.clone()
    kv1 = ra.PagedKV(k1, v1, i32(lay.block_table, device), *sc)
    o1, l1 = ra.append_write(q, k_new, v_new, cu_t, ctx_t, kv1, max(T), max_kv, SCALE,
                             want_lse=True, cos_sin=tab)
    # separate: rotated write, then append on the oracle-rotated queries
    pos = np.concatenate([np.arange(c, c + t) for c, t in zip(ctx, T)]).astype(np.int32)
    q_rot = oracle.rope(bits(q), pos, table)
    k2, v2 = k.clone(), v.clone()
    kv2 = ra.PagedKV(k2, v2, i32(lay.block_table, device), *sc)
    ra.kv_page_write(k_new, v_new, cu_t, ctx_t, kv2, max(T), max_kv, cos_sin=tab)
    o2, l2 = ra.append(from_bits(q_rot, device), cu_t, ctx_t, kv2, max(T), max_kv, SCALE,
                       want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(k1, k2) and torch.equal(v1, v2), "pools differ"
    assert torch.equal(o1, o2) and torch.equal(l1, l2), "fused rotated append differs"
    if fp8:
        ref, ref_lse = oracle.append_fp8(q_rot, cu, ctx, bits(k1), bits(v1), ks, vs,
                                         lay.block_table, SCALE)
    else:
        ref, ref_lse = oracle.append(q_rot, cu, ctx, bits(k1), bits(v1), lay.block_table, SCALE)
    assert_attn_close(o1.cpu().numpy(), ref, f"append_write_rope G={Hq // Hkv} fp8={fp8}")
    np.testing.assert_allclose(l1.cpu().numpy(), ref_lse, atol=APPEND_LSE_ATOL, rtol=0)
