"""GPU parity at non-positive softmax scales (through the C ABI) against the fp64
CPU oracle.

The ABI accepts any finite scale. A zero scale makes every attended key equally
likely (out = the mean of the attended V rows, lse = ln of their count, a
closed form); a negative scale reverses the order of the scores. Append and
the mixed step run a kernel variant of their own when the scale is not
positive (scores are scaled before the exponent instead of inside it), so
these cases exercise code the positive-scale tests do not reach.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2603_18815_amd as ra
import synth
from tests.gpu_util import APPEND_LSE_ATOL, assert_attn_close, attn_stats, bits

pytestmark = pytest.mark.gpu
SCALES = [0.0, -0.7 / math.sqrt(128)]


def i32(x, dev):
    return torch.as_tensor(np.ascontiguousarray(np.asarray(x, np.int32)), device=dev)


def say(msg):
    print(f"[gpu-test] {msg}", flush=True)


def pool(seed, row_tokens, Hkv, dev):
    rng = np.random.default_rng(seed)
    lay = synth.make_layout(rng, row_tokens)
    gen = synth.value_generator(seed, dev)
    k = synth.randn_bf16((lay.num_pages, Hkv, 16, 128), gen, dev)
    v = synth.randn_bf16((lay.num_pages, Hkv, 128, 16), gen, dev)
    return lay, k, v, gen


@pytest.mark.parametrize("scale", SCALES)
def test_decode_nonpositive_scale(device, scale):
    lens = [1, 17, 300, 1000]
    Hq, Hkv = 8, 2
    say(f"decode scale={scale}")
    lay, k, v, gen = pool(11, lens, Hkv, device)
    q = synth.randn_bf16((len(lens), Hq, 128), gen, device)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device))
    out, lse = ra.decode(q, kv, i32(lens, device), max(lens), scale, want_lse=True)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.decode(bits(q), bits(k), bits(v), lay.block_table, lens, scale)
    assert_attn_close(out.cpu().numpy(), ref, f"decode scale={scale}")
    np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, atol=1e-4, rtol=0)
    if scale == 0.0:
        # closed form: uniform weights
        np.testing.assert_allclose(lse.cpu().numpy(),
                                   np.log(np.array(lens, np.float64))[:, None].repeat(Hq, 1),
                                   atol=1e-5, rtol=0)


@pytest.mark.parametrize("scale", SCALES)
@pytest.mark.parametrize("fp8", [False, True])
def test_append_nonpositive_scale(device, scale, fp8):
    ctx, T = [0, 17, 300, 40], [5, 64, 130, 300]
    Hq, Hkv = 32, 8
    say(f"append scale={scale} fp8={fp8}")
    lens = [c + n for c, n in zip(ctx, T)]
    lay, k, v, gen = pool(12, lens, Hkv, device)
    cu = np.concatenate([[0], np.cumsum(T)]).astype(np.int32)
    q = synth.randn_bf16((int(cu[-1]), Hq, 128), gen, device)
    if fp8:
        ks, vs = 0.05, 0.04
        k = synth.randn_fp8_codes(tuple(k.shape), gen, device, ks)
        v = synth.randn_fp8_codes(tuple(v.shape), gen, device, vs)
        kv = ra.PagedKV(k, v, i32(lay.block_table, device), ks, vs)
    else:
        kv = ra.PagedKV(k, v, i32(lay.block_table, device))
    out, lse = ra.append(q, i32(cu, device), i32(ctx, device), kv, max(T), max(lens), scale,
                         want_lse=True)
    torch.cuda.synchronize()
    if fp8:
        ref, ref_lse = oracle.append_fp8(bits(q), cu, ctx, bits(k), bits(v), ks, vs,
                                         lay.block_table, scale)
    else:
        ref, ref_lse = oracle.append(bits(q), cu, ctx, bits(k), bits(v), lay.block_table, scale)
    assert_attn_close(out.cpu().numpy(), ref, f"append scale={scale} fp8={fp8}")
    np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, atol=APPEND_LSE_ATOL, rtol=0)


@pytest.mark.parametrize("scale", SCALES)
def test_mixed_nonpositive_scale(device, scale):
    """Decode and append rows in one launch: the append part bitwise equals the
    append call, the decode part meets the oracle."""
    w = synth.mixed_workload(13, 20, 32, 8, 0.35,
                             lambda r, n: synth.uniform_int(r, n, 0, 1200),
                             lambda r, n: synth.uniform_int(r, n, 1, 260),
                             "small mixed, non-positive scale")
    say(f"mixed scale={scale}: {w.decode_rows.size} decode rows, {w.append_rows.size} append")
    t = synth.make_tensors(w, device)
    kd = ra.PagedKV(t.k_pool, t.v_pool, i32(w.decode_table(), device))
    ka = ra.PagedKV(t.k_pool, t.v_pool, i32(w.append_table(), device))
    mk, mq = int(w.kv_lens.max()), int(w.q_lens.max())
    mka = int((w.ctx_lens + w.q_lens).max())
    cu, ctx = i32(w.cu_q(), device), i32(w.ctx_lens, device)
    od, oa, ld, la = ra.mixed(t.q_decode, kd, i32(w.kv_lens, device), t.q_append, cu, ctx, ka,
                              mk, mq, mka, scale, want_lse=True)
    sa, sla = ra.append(t.q_append, cu, ctx, ka, mq, mka, scale, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(oa, sa) and torch.equal(la, sla), "append part differs from append()"
    ref_d, ref_ld = oracle.decode(bits(t.q_decode), bits(t.k_pool), bits(t.v_pool),
                                  w.decode_table(), w.kv_lens, scale)
    assert_attn_close(od.cpu().numpy(), ref_d, f"mixed decode scale={scale}")
    np.testing.assert_allclose(ld.cpu().numpy(), ref_ld, atol=1e-4, rtol=0)


SHARP = 16.0 / math.sqrt(128)   # scores of standard deviation ~16 (natural units)


def assert_sharp_close(gpu, ref, vmax, what):
    """Append at a sharp softmax. The kernel rounds each weight to bf16
    (relative error <= 2^-9) before both P·V and the normaliser, so an output
    moves by at most sum_j |p~_j - p_j| |v_j - out| <= 2^-8 max|v| (the
    p~ - p sum to zero); the rel-L2 bound of the other tests still holds."""
    g = np.asarray(gpu, np.float64)
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    max_abs, rel = attn_stats(g, ref)
    print(f"[parity] {what}: max_abs={max_abs:.3e} rel_l2={rel:.3e} bound={2.0**-8 * vmax:.3e}", flush=True)
    assert max_abs <= max(2.0 ** -8 * vmax, 1e-2) and rel <= 5e-3, (what, max_abs, rel)


@pytest.mark.parametrize("kind", ["decode", "append", "append_fp8", "mixed"])
def test_sharp_softmax_moves_the_running_max(device, kind):
    """A large scale, so that the append kernel's rescaling path runs: its
    weights are taken against a running maximum kept until they would exceed
    2^14, and random inputs at the usual scale rarely get there. On the append
    inputs below, 38 % of the (query, head) pairs see a later pair of keys
    whose maximum score exceeds the running one by more than 14 (base 2),
    7,369 times in all (counted on the CPU from the same seeded inputs)."""
    say(f"sharp softmax {kind}")
    Hq, Hkv = 32, 8
    if kind == "decode":
        lens = [1, 33, 700, 2100]
        lay, k, v, gen = pool(21, lens, Hkv, device)
        q = synth.randn_bf16((len(lens), Hq, 128), gen, device)
        kv = ra.PagedKV(k, v, i32(lay.block_table, device))
        out, lse = ra.decode(q, kv, i32(lens, device), max(lens), SHARP, want_lse=True)
        torch.cuda.synchronize()
        ref, ref_lse = oracle.decode(bits(q), bits(k), bits(v), lay.block_table, lens, SHARP)
        assert_attn_close(out.cpu().numpy(), ref, "decode, sharp")
        np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, atol=1e-4, rtol=0)
    elif kind in ("append", "append_fp8"):
        ctx, T = [0, 40, 900, 1500], [70, 300, 129, 40]
        lens = [c + n for c, n in zip(ctx, T)]
        lay, k, v, gen = pool(22, lens, Hkv, device)
        cu = np.concatenate([[0], np.cumsum(T)]).astype(np.int32)
        q = synth.randn_bf16((int(cu[-1]), Hq, 128), gen, device)
        if kind == "append_fp8":
            ks, vs = 0.05, 0.04
            k = synth.randn_fp8_codes(tuple(k.shape), gen, device, ks)
            v = synth.randn_fp8_codes(tuple(v.shape), gen, device, vs)
            kv = ra.PagedKV(k, v, i32(lay.block_table, device), ks, vs)
        else:
            kv = ra.PagedKV(k, v, i32(lay.block_table, device))
        out, lse = ra.append(q, i32(cu, device), i32(ctx, device), kv, max(T), max(lens), SHARP,
                             want_lse=True)
        torch.cuda.synchronize()
        if kind == "append_fp8":
            ref, ref_lse = oracle.append_fp8(bits(q), cu, ctx, bits(k), bits(v), ks, vs,
                                             lay.block_table, SHARP)
            vmax = float(np.abs(oracle.e4m3_decode(bits(v))).max()) * vs
        else:
            ref, ref_lse = oracle.append(bits(q), cu, ctx, bits(k), bits(v), lay.block_table, SHARP)
            vmax = float(v.float().abs().max())
        assert_sharp_close(out.cpu().numpy(), ref, vmax, f"{kind}, sharp")
        np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, atol=APPEND_LSE_ATOL, rtol=0)
    else:
        w = synth.mixed_workload(23, 20, 32, 8, 0.35,
                                 lambda r, n: synth.uniform_int(r, n, 0, 1500),
                                 lambda r, n: synth.uniform_int(r, n, 1, 300),
                                 "small mixed, sharp softmax")
        t = synth.make_tensors(w, device)
        kd = ra.PagedKV(t.k_pool, t.v_pool, i32(w.decode_table(), device))
        ka = ra.PagedKV(t.k_pool, t.v_pool, i32(w.append_table(), device))
        mk, mq = int(w.kv_lens.max()), int(w.q_lens.max())
        mka = int((w.ctx_lens + w.q_lens).max())
        cu, ctx = i32(w.cu_q(), device), i32(w.ctx_lens, device)
        od, oa, ld, la = ra.mixed(t.q_decode, kd, i32(w.kv_lens, device), t.q_append, cu, ctx, ka,
                                  mk, mq, mka, SHARP, want_lse=True)
        sa, sla = ra.append(t.q_append, cu, ctx, ka, mq, mka, SHARP, want_lse=True)
        torch.cuda.synchronize()
        assert torch.equal(oa, sa) and torch.equal(la, sla), "append part differs from append()"
        ref_d, ref_ld = oracle.decode(bits(t.q_decode), bits(t.k_pool), bits(t.v_pool),
                                      w.decode_table(), w.kv_lens, SHARP)
        assert_attn_close(od.cpu().numpy(), ref_d, "mixed decode, sharp")
        np.testing.assert_allclose(ld.cpu().numpy(), ref_ld, atol=1e-4, rtol=0)
        ref_a, ref_la = oracle.append(bits(t.q_append), w.cu_q(), w.ctx_lens, bits(t.k_pool),
                                      bits(t.v_pool), w.append_table(), SHARP)
        assert_sharp_close(oa.cpu().numpy(), ref_a, float(t.v_pool.float().abs().max()), "mixed append, sharp")
        np.testing.assert_allclose(la.cpu().numpy(), ref_la, atol=APPEND_LSE_ATOL, rtol=0)
