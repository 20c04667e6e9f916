"""GPU parity of fp8 (OCP E4M3) KV pools (through the C ABI) against the fp64 CPU oracle.

Page writes into fp8 pools must store bit-exactly the codes the oracle's
quantizer gives (every bf16 value, NaN and infinities included, at several
scales); the gather must return the stored codes bit-exactly. Decode over fp8
pools is checked against the oracle's attention over the dequantized values at
the attention tolerance of tests.gpu_util.
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


def fp8_pool(seed, row_tokens, Hkv, dev, scale):
    """A shuffled page layout for the rows and fp8 pools of N(0,1) / scale codes."""
    rng = np.random.default_rng(seed)
    lay = synth.make_layout(rng, row_tokens)
    gen = synth.value_generator(seed, dev)
    k = synth.randn_fp8_codes((lay.num_pages, Hkv, 16, 128), gen, dev, scale)
    v = synth.randn_fp8_codes((lay.num_pages, Hkv, 128, 16), gen, dev, scale)
    return lay, k, v, gen


@pytest.mark.parametrize("k_scale,v_scale", [(1.0, 1.0), (0.0371, 13.5), (2.0 ** -6, 3e-3)])
def test_fp8_page_write_every_bf16_value_bitexact(device, k_scale, v_scale):
    """All 65536 bf16 bit patterns written into fp8 pools at ragged positions: the
    whole pools must equal the oracle's (quantized tokens in place, nothing else
    changed), and the gather must return the codes."""
    say(f"fp8 page write, scales {k_scale} / {v_scale}")
    Hkv = 2
    allbits = np.arange(1 << 16, dtype=np.uint16)
    rng = np.random.default_rng(1)
    vals = allbits.reshape(256, Hkv, 128)                     # 256 tokens
    k_new = vals
    v_new = vals[rng.permutation(256)]
    new = [37, 1, 100, 118]                                  # ragged, 256 tokens in total
    old = [5, 16, 0, 33]
    total = [o + n for o, n in zip(old, new)]
    lay, k, v, gen = fp8_pool(2, total, Hkv, device, 0.25)
    cu = np.concatenate([[0], np.cumsum(new)]).astype(np.int32)
    kp0, vp0 = bits(k), bits(v)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device), k_scale, v_scale)
    tk = torch.from_numpy(k_new.view(np.int16).copy()).view(torch.bfloat16).to(device)
    tv = torch.from_numpy(v_new.view(np.int16).copy()).view(torch.bfloat16).to(device)
    ra.kv_page_write(tk, tv, i32(cu, device), i32(old, device), kv, max(new), max(total))
    cu_out = np.concatenate([[0], np.cumsum(total)]).astype(np.int32)
    ko, vo = ra.kv_page_gather(kv, i32(total, device), i32(cu_out, device))
    torch.cuda.synchronize()
    kx, vx = oracle.page_write_fp8(k_new, v_new, cu, old, lay.block_table, kp0, vp0, k_scale,
                                   v_scale)
    np.testing.assert_array_equal(bits(k), kx)
    np.testing.assert_array_equal(bits(v), vx)
    kg, vg = oracle.page_gather_u8(kx, vx, lay.block_table, total, cu_out)
    np.testing.assert_array_equal(bits(ko), kg)
    np.testing.assert_array_equal(bits(vo), vg)
    q = oracle.quantize(k_new, k_scale)
    assert (q == 0x7F).any() and ((q == 0x7E) | (q == 0xFE)).any()   # NaN and saturation seen


@pytest.mark.parametrize("Hq,Hkv", [(32, 8), (8, 8), (16, 1), (8, 2), (32, 1)])
def test_fp8_decode_vs_oracle(device, Hq, Hkv):
    lens = [1, 15, 16, 17, 31, 32, 33, 300, 1000, 2049, 4100]
    ks, vs = 2.0 ** -5, 0.0625
    say(f"fp8 decode Hq={Hq} Hkv={Hkv}")
    lay, k, v, gen = fp8_pool(Hq + Hkv, lens, Hkv, device, ks)
    q = synth.randn_bf16((len(lens), Hq, 128), gen, device)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device), ks, vs)
    out, lse = ra.decode(q, kv, i32(lens, device), max(lens), SCALE, want_lse=True)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.decode_fp8(bits(q), bits(k), bits(v), ks, vs, lay.block_table, lens,
                                     SCALE)
    assert_attn_close(out.cpu().numpy(), ref, f"fp8 decode G={Hq // Hkv}")
    np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, atol=1e-4, rtol=0)


def test_fp8_decode_one_key_returns_each_code_exactly(device):
    """With one key the output is v_scale times that key's dequantized V row, exactly:
    every finite E4M3 code passes through the exact conversion to bf16."""
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], np.uint8)
    rows = (len(codes) + 127) // 128
    Hq = Hkv = 1
    lay, k, v, gen = fp8_pool(4, [1] * rows, Hkv, device, 1.0)
    vc = np.resize(codes, rows * 128).reshape(rows, 128)
    for r in range(rows):
        v[int(lay.block_table[r, 0]), 0, :, 0] = torch.from_numpy(vc[r]).to(device)
    q = synth.randn_bf16((rows, Hq, 128), gen, device)
    vs = 0.75
    kv = ra.PagedKV(k, v, i32(lay.block_table, device), 0.5, vs)
    out, lse = ra.decode(q, kv, i32([1] * rows, device), 1, SCALE, want_lse=True)
    torch.cuda.synchronize()
    want = (oracle.e4m3_decode(vc).astype(np.float32) * np.float32(vs)).astype(np.float32)
    np.testing.assert_array_equal(out.cpu().numpy()[:, 0, :], want)


def test_fp8_decode_poison_and_determinism(device):
    """E4M3 NaN codes in pages no row owns and past each row's end are bitwise
    invisible; repeated calls agree bitwise."""
    lens = [3, 16, 17, 200, 513]
    lay, k, v, gen = fp8_pool(6, lens, 8, device, 0.05)
    q = synth.randn_bf16((len(lens), 32, 128), gen, device)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device), 0.05, 0.3)
    args = (q, kv, i32(lens, device), max(lens), SCALE)
    a, la = ra.decode(*args, want_lse=True)
    b, lb = ra.decode(*args, want_lse=True)
    synth.poison_unowned(k, v, lay, lens=lens)
    c, lc = ra.decode(*args, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(la, lb)
    assert torch.equal(a, c) and torch.equal(la, lc)


def test_fp8_shared_prefix_decode_vs_oracle(device):
    Hq, Hkv = 32, 8
    rng = np.random.default_rng(8)
    sizes = [8, 3]
    pre = np.array([45, 20], np.int64) * 16
    suffix = rng.integers(1, 600, size=sum(sizes))
    lay = synth.shared_prefix_layout(rng, sizes, pre, suffix)
    gen = synth.value_generator(8, device)
    ks, vs = 0.02, 0.5
    k = synth.randn_fp8_codes((lay.num_pages, Hkv, 16, 128), gen, device, ks)
    v = synth.randn_fp8_codes((lay.num_pages, Hkv, 128, 16), gen, device, ks)
    q = synth.randn_bf16((len(suffix), Hq, 128), gen, device)
    lens = lay.row_tokens.astype(np.int32)
    gs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device), ks, vs)
    out, lse = ra.decode_shared_prefix(q, kv, i32(lens, device), i32(gs, device),
                                       i32(pre.astype(np.int32), device), max(sizes),
                                       int(pre.max()), int(lens.max()), SCALE, want_lse=True)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.decode_fp8(bits(q), bits(k), bits(v), ks, vs, lay.block_table, lens,
                                     SCALE)
    assert_attn_close(out.cpu().numpy(), ref, "fp8 shared-prefix decode")
    np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, atol=1e-4, rtol=0)


def test_fp8_decode_qwen3_workload_sampled(device):
    """The B=64 Qwen3-8B decode workload with an fp8 pool, sampled rows vs the oracle."""
    w = synth.config(2)
    say(f"fp8 decode {w.name}")
    ks, vs = 2.0 ** -5, 2.0 ** -5
    lay = w.layout
    gen = synth.value_generator(22, device)
    k = synth.randn_fp8_codes((lay.num_pages, w.Hkv, 16, 128), gen, device, ks)
    v = synth.randn_fp8_codes((lay.num_pages, w.Hkv, 128, 16), gen, device, vs)
    q = synth.randn_bf16((w.kv_lens.size, w.Hq, 128), gen, device)
    bt = w.decode_table()
    kv = ra.PagedKV(k, v, i32(bt, device), ks, vs)
    out, lse = ra.decode(q, kv, i32(w.kv_lens, device), int(w.kv_lens.max()), SCALE,
                         want_lse=True)
    torch.cuda.synchronize()
    rows = sample_rows(w.kv_lens, 5, seed=2)
    kc, vc, btc = compact_rows(k, v, bt[rows], w.kv_lens[rows])
    ref, ref_lse = oracle.decode_fp8(bits(q[torch.as_tensor(rows, device=device)]), kc, vc, ks,
                                     vs, btc, w.kv_lens[rows], SCALE)
    sel = torch.as_tensor(rows, device=device)
    assert_attn_close(out[sel].cpu().numpy(), ref, "fp8 decode workload 2 sampled")
    np.testing.assert_allclose(lse[sel].cpu().numpy(), ref_lse, atol=1e-4, rtol=0)


@pytest.mark.parametrize("Hq,Hkv", [(32, 8), (16, 1), (64, 8)])
def test_fp8_append_vs_oracle(device, Hq, Hkv):
    ctx = [0, 1, 15, 16, 17, 100, 300, 2000]
    T = [5, 64, 1, 63, 65, 200, 130, 17]
    ks, vs = 2.0 ** -5, 0.04
    say(f"fp8 append Hq={Hq} Hkv={Hkv}")
    lay, k, v, gen = fp8_pool(Hq * 5 + Hkv, [c + t for c, t in zip(ctx, T)], Hkv, device, ks)
    cu = np.concatenate([[0], np.cumsum(T)]).astype(np.int32)
    q = synth.randn_bf16((int(cu[-1]), Hq, 128), gen, device)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device), ks, vs)
    out, lse = ra.append(q, i32(cu, device), i32(ctx, device), kv, max(T),
                         max(c + t for c, t in zip(ctx, T)), SCALE, want_lse=True)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.append_fp8(bits(q), cu, ctx, bits(k), bits(v), ks, vs,
                                     lay.block_table, SCALE)
    assert_attn_close(out.cpu().numpy(), ref, f"fp8 append G={Hq // Hkv}")
    np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, atol=APPEND_LSE_ATOL, rtol=0)


def test_fp8_append_poison_invisible(device):
    ctx, T = [0, 17, 250, 1000], [33, 100, 64, 7]
    lay, k, v, gen = fp8_pool(77, [c + t for c, t in zip(ctx, T)], 8, device, 0.05)
    cu = np.concatenate([[0], np.cumsum(T)]).astype(np.int32)
    q = synth.randn_bf16((int(cu[-1]), 32, 128), gen, device)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device), 0.05, 0.2)
    args = (q, i32(cu, device), i32(ctx, device), kv, max(T), 1007, SCALE)
    a, la = ra.append(*args, want_lse=True)
    synth.poison_unowned(k, v, lay)
    b, lb = ra.append(*args, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(la, lb)


def test_fp8_mixed_step_vs_oracle(device):
    """Decode rows and append rows of one step over one fp8 pool, in one launch."""
    w = synth.mixed_workload(31, 24, 32, 8, 0.35,
                             lambda r, n: synth.uniform_int(r, n, 0, 1500),
                             lambda r, n: synth.uniform_int(r, n, 1, 300), "small fp8 mixed")
    ks, vs = 2.0 ** -5, 0.05
    gen = synth.value_generator(31, device)
    k = synth.randn_fp8_codes((w.layout.num_pages, 8, 16, 128), gen, device, ks)
    v = synth.randn_fp8_codes((w.layout.num_pages, 8, 128, 16), gen, device, ks)
    qd = synth.randn_bf16((w.kv_lens.size, 32, 128), gen, device)
    qa = synth.randn_bf16((int(w.q_lens.sum()), 32, 128), gen, device)
    kd = ra.PagedKV(k, v, i32(w.decode_table(), device), ks, vs)
    ka = ra.PagedKV(k, v, i32(w.append_table(), device), ks, vs)
    mq, mka = int(w.q_lens.max()), int((w.ctx_lens + w.q_lens).max())
    od, oa, ld, la = ra.mixed(qd, kd, i32(w.kv_lens, device), qa, i32(w.cu_q(), device),
                              i32(w.ctx_lens, device), ka, int(w.kv_lens.max()), mq, mka, SCALE,
                              want_lse=True)
    sa, _ = ra.append(qa, i32(w.cu_q(), device), i32(w.ctx_lens, device), ka, mq, mka, SCALE)
    torch.cuda.synchronize()
    assert torch.equal(oa, sa), "fp8 mixed append part differs from append()"
    ref_d, _ = oracle.decode_fp8(bits(qd), bits(k), bits(v), ks, vs, w.decode_table(),
                                 w.kv_lens, SCALE)
    assert_attn_close(od.cpu().numpy(), ref_d, "fp8 mixed decode rows")
    ref_a, _ = oracle.append_fp8(bits(qa), w.cu_q(), w.ctx_lens, bits(k), bits(v), ks, vs,
                                 w.append_table(), SCALE)
    assert_attn_close(oa.cpu().numpy(), ref_a, "fp8 mixed append rows")
