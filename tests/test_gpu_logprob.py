"""GPU parity of token_logprob (through the C ABI) against the fp64 CPU oracle.

Tolerance: the library accumulates each logit in fp32 over D products of
exactly-widened bf16 values (the products are exact) and uses the hardware
exp2/log2 (about 1 ulp); the oracle is fp64. Rounding in a sum of D terms
behaves like a random walk, about sqrt(D) * 2^-24 * |terms| ~ 1e-6 for the
inputs here (logits of order 1-10, D <= 4096), against a loose worst case of
D * 2^-24 * sum_k |h_k W_vk|. Every log-probability and lse must agree within
1e-4 absolute; out-of-range targets must give NaN.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2603_18815_amd as ra
import synth
from tests.gpu_util import bits

pytestmark = pytest.mark.gpu
ATOL = 1e-4


def say(msg):
    print(f"[gpu-test] {msg}", flush=True)


def inputs(seed, N, V, D, dev, w_scale=None):
    """h ~ N(0,1), W ~ N(0, 1/D) (logits of order 1), both rounded to bf16."""
    gen = synth.value_generator(seed, dev)
    h = synth.randn_bf16((N, D), gen, dev)
    W = synth.randn_bf16((V, D), gen, dev)
    s = 1.0 / math.sqrt(D) if w_scale is None else w_scale
    W = (W.float() * s).to(torch.bfloat16)
    return h, W


def check(lp, ls, ref_lp, ref_ls, what):
    lp, ls = lp.cpu().numpy().astype(np.float64), ls.cpu().numpy().astype(np.float64)
    ok = ~np.isnan(ref_lp)
    assert np.all(np.isnan(lp[~ok])), f"{what}: out-of-range targets must give NaN"
    err_lp = float(np.abs(lp[ok] - ref_lp[ok]).max()) if ok.any() else 0.0
    err_ls = float(np.abs(ls - ref_ls).max())
    print(f"[parity] {what}: max|dlogp|={err_lp:.2e} max|dlse|={err_ls:.2e}", flush=True)
    assert err_lp <= ATOL and err_ls <= ATOL, (what, err_lp, err_ls)


@pytest.mark.parametrize("N,V,D,scale", [
    (70, 1000, 128, 1.0),    # two token blocks (ragged), a ragged last vocabulary chunk
    (5, 257, 192, 0.7),      # temperature scale, vocabulary of 2 chunks + 1 row
    (1, 1, 64, 1.0),         # a single vocabulary entry: logp = 0
    (130, 4096, 256, 1.0),   # three token blocks, 32 chunks (4 per XCD)
    # from N = 512 on: 384 x 256 tiles through the LDS ring
    (512, 1000, 128, 0.7),   # two token blocks, a ragged last 384-row chunk
    (600, 5000, 256, 1.0),   # a ragged third token block
    (2000, 700, 64, 1.0),    # D = 64: two steps, fewer than the ring's stages
    (1024, 3000, 192, 1.3),  # D = 192: six steps (the ring wraps once, ragged)
    (520, 1, 64, 1.0),       # one vocabulary entry in a 384-row chunk: logp = 0
])
def test_token_logprob_vs_oracle(device, N, V, D, scale):
    say(f"token_logprob N={N} V={V} D={D} scale={scale}")
    h, W = inputs(N + V + D, N, V, D, device)
    rng = np.random.default_rng(N + V)
    t = rng.integers(0, V, size=N).astype(np.int32)
    if N >= 5:
        t[:4] = [0, V - 1, -1, V]           # first and last id, two out of range
    lp, ls = ra.token_logprob(h, W, torch.as_tensor(t, device=device), scale, want_lse=True)
    torch.cuda.synchronize()
    ref_lp, ref_ls = oracle.token_logprob(bits(h), bits(W), t, scale)
    check(lp, ls, ref_lp, ref_ls, f"N={N} V={V} D={D}")
    if V == 1:
        # one entry: logp = 0 up to the rounding of z - lse (targets out of range are NaN)
        valid = ~np.isnan(ref_lp)
        assert np.all(np.abs(lp.cpu().numpy()[valid]) <= 1e-6)


def test_token_logprob_peaked_and_flat(device):
    """Large logits (a peaked distribution) and zero hidden states (uniform)."""
    N, V, D = 40, 3000, 128
    h, W = inputs(5, N, V, D, device, w_scale=0.5)     # logits of order 5-20
    h[:8] = 0                                           # uniform rows
    t = torch.arange(N, dtype=torch.int32, device=device) * 71 % V
    lp, ls = ra.token_logprob(h, W, t, 1.0, want_lse=True)
    torch.cuda.synchronize()
    ref_lp, ref_ls = oracle.token_logprob(bits(h), bits(W), t.cpu().numpy(), 1.0)
    check(lp, ls, ref_lp, ref_ls, "peaked / flat")
    np.testing.assert_allclose(lp[:8].cpu().numpy(), -math.log(V), atol=1e-5, rtol=0)


@pytest.mark.parametrize("N", [4, 520])
def test_token_logprob_logits_near_1000(device, N):
    """Logits up to ~1,016, far past where exp overflows fp32 unless the
    maximum is taken out first: W[v] = (1000 - 4 (v % 97), small integer) and
    h[n] = (1, n % 5 - 2), all exact in bf16, so every logit is an exact
    integer in fp32 too. N = 4 runs the partial kernel, N = 520 the tiled one,
    both layouts of W. The remaining error is fp32 rounding of values near
    1,000 (and near 1,443 in base-2 units): a few 1e-4, so this test allows
    5e-4 absolute."""
    say(f"token_logprob logits near 1000 N={N}")
    V, D = 700, 64
    v = np.arange(V)
    Wf = np.zeros((V, D), np.float32)
    Wf[:, 0] = 1000 - 4 * (v % 97)
    Wf[:, 1] = (v * 7) % 17 - 8
    hf = np.zeros((N, D), np.float32)
    hf[:, 0] = 1.0
    hf[:, 1] = np.arange(N) % 5 - 2
    W = torch.from_numpy(Wf).to(torch.bfloat16).to(device)
    h = torch.from_numpy(hf).to(torch.bfloat16).to(device)
    assert torch.equal(W.float().cpu(), torch.from_numpy(Wf)) and torch.equal(h.float().cpu(), torch.from_numpy(hf))
    t = torch.from_numpy((np.arange(N) * 37 % V).astype(np.int32)).to(device)
    lp, ls = ra.token_logprob(h, W, t, 1.0, want_lse=True)
    lq, lsq = ra.token_logprob_packed(h, ra.token_logprob_pack_weight(W), V, t, 1.0, want_lse=True)
    torch.cuda.synchronize()
    ref_lp, ref_ls = oracle.token_logprob(bits(h), bits(W), t.cpu().numpy(), 1.0)
    assert np.all(ref_ls > 999.0)
    for a, b, what in ((lp, ls, "row-major"), (lq, lsq, "packed")):
        a, b = a.cpu().numpy().astype(np.float64), b.cpu().numpy().astype(np.float64)
        assert np.all(np.isfinite(a)) and np.all(np.isfinite(b)), what
        err_lp, err_ls = float(np.abs(a - ref_lp).max()), float(np.abs(b - ref_ls).max())
        print(f"[parity] logits near 1000 N={N} {what}: max|dlogp|={err_lp:.2e} max|dlse|={err_ls:.2e}", flush=True)
        assert err_lp <= 5e-4 and err_ls <= 5e-4, (what, err_lp, err_ls)
    assert torch.equal(lp, lq) and torch.equal(ls, lsq)


def test_token_logprob_deterministic(device):
    N, V, D = 64, 5000, 256
    h, W = inputs(9, N, V, D, device)
    t = torch.randint(0, V, (N,), dtype=torch.int32, device=device,
                      generator=synth.value_generator(9, device))
    a, la = ra.token_logprob(h, W, t, 1.0, want_lse=True)
    b, lb = ra.token_logprob(h, W, t, 1.0, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(la, lb)


def test_token_logprob_qwen3_lm_head(device):
    """The Qwen3-8B LM-head shape (V = 151936, D = 4096) for a decode batch of 64
    tokens, every token against the oracle."""
    N, V, D = 64, 151936, 4096
    say(f"token_logprob Qwen3-8B LM head N={N}")
    h, W = inputs(8, N, V, D, device)
    t = torch.randint(0, V, (N,), dtype=torch.int32, device=device,
                      generator=synth.value_generator(8, device))
    lp, ls = ra.token_logprob(h, W, t, 1.0, want_lse=True)
    torch.cuda.synchronize()
    ref_lp, ref_ls = oracle.token_logprob(bits(h), bits(W), t.cpu().numpy(), 1.0)
    check(lp, ls, ref_lp, ref_ls, "Qwen3-8B LM head, 64 tokens")


def packed_layout(W_bits, V, D):
    """The packed LM-head layout restated from its definition: with T tiles of
    32 rows (V rounded up to a multiple of 384), 16-byte unit
    ((s * T + tile) * 4 + u) * 64 + lane holds row 32 tile + lane % 32, dims
    64 s + 32 (lane / 32) + 8 u + 0..7; rows past V are zeros."""
    Vp = (V + 383) // 384 * 384
    Wz = np.zeros((Vp, D), np.uint16)
    Wz[:V] = W_bits
    x = Wz.reshape(Vp // 32, 32, D // 64, 2, 4, 8)      # tile, row, s, half, u, e
    x = x.transpose(2, 0, 4, 3, 1, 5)                   # s, tile, u, half, row, e
    return x.reshape(-1)                                # lane = 32 half + row


@pytest.mark.parametrize("V,D", [(200, 128), (128, 64), (1, 192), (1000, 256)])
def test_pack_weight_layout(device, V, D):
    """The packed copy is bit-exactly the documented permutation of W."""
    say(f"token_logprob_pack_weight V={V} D={D}")
    _, W = inputs(V + D, 1, V, D, device)
    Wp = ra.token_logprob_pack_weight(W)
    torch.cuda.synchronize()
    assert Wp.numel() == (V + 383) // 384 * 384 * D
    assert np.array_equal(bits(Wp), packed_layout(bits(W), V, D))


@pytest.mark.parametrize("N,V,D,scale", [
    (70, 1000, 128, 1.0),
    (5, 257, 192, 0.7),
    (1, 1, 64, 1.0),
    (130, 4096, 256, 1.0),
    (64, 3001, 320, 1.3),
    (512, 1000, 128, 0.7),
    (600, 5000, 256, 1.0),
    (2000, 700, 64, 1.0),
    (1024, 3000, 192, 1.3),
])
def test_token_logprob_packed_matches(device, N, V, D, scale):
    """token_logprob_packed gives bitwise the row-major results, and both meet
    the oracle."""
    say(f"token_logprob_packed N={N} V={V} D={D} scale={scale}")
    h, W = inputs(N + V + D + 1, N, V, D, device)
    rng = np.random.default_rng(N + V + 1)
    t = rng.integers(0, V, size=N).astype(np.int32)
    if N >= 5:
        t[:4] = [0, V - 1, -1, V]
    tt = torch.as_tensor(t, device=device)
    Wp = ra.token_logprob_pack_weight(W)
    lp, ls = ra.token_logprob(h, W, tt, scale, want_lse=True)
    lp2, ls2 = ra.token_logprob_packed(h, Wp, V, tt, scale, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(lp.isnan(), lp2.isnan())
    assert torch.equal(torch.nan_to_num(lp), torch.nan_to_num(lp2)) and torch.equal(ls, ls2)
    ref_lp, ref_ls = oracle.token_logprob(bits(h), bits(W), t, scale)
    check(lp2, ls2, ref_lp, ref_ls, f"packed N={N} V={V} D={D}")


@pytest.mark.parametrize("N", [64, 1024, 4000])
def test_token_logprob_packed_qwen3_lm_head(device, N):
    """The Qwen3-8B LM head at the benchmark's batch sizes and at 4,000 tokens
    (16 token blocks, the last one ragged; ~25 rounds of tiles): packed and
    row-major bitwise equal; 16 sampled tokens plus the first and the last
    against the oracle."""
    V, D = 151936, 4096
    say(f"token_logprob_packed Qwen3-8B LM head N={N}")
    h, W = inputs(80 + N, N, V, D, device)
    t = torch.randint(0, V, (N,), dtype=torch.int32, device=device,
                      generator=synth.value_generator(80 + N, device))
    Wp = ra.token_logprob_pack_weight(W)
    lp, ls = ra.token_logprob(h, W, t, 1.0, want_lse=True)
    lp2, ls2 = ra.token_logprob_packed(h, Wp, V, t, 1.0, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(lp, lp2) and torch.equal(ls, ls2)
    del Wp
    pick = np.array(sorted(set(np.random.default_rng(N).choice(N, size=16, replace=False)) | {0, N - 1}))
    ref_lp, ref_ls = oracle.token_logprob(bits(h)[pick], bits(W), t.cpu().numpy()[pick], 1.0)
    check(lp2[pick], ls2[pick], ref_lp, ref_ls, f"packed Qwen3-8B LM head, N={N} ({pick.size} sampled)")
