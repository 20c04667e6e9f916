"""Pins of the fp64 CPU oracle against facts that do not come from the oracle.

The paper prints no attention values, so the oracle is pinned by
  * a library routine: torch's fp64 scaled_dot_product_attention with an
    explicit boolean mask and its own grouped-query head mapping;
  * a dense brute force that reads the pages through numpy subscripts;
  * closed forms (one key, identical keys, two keys) and hand-worked fixtures
    under tests/golden/;
  * invariants (page permutation, causality, append with T=1 == decode, key
    shift, value affinity, group consistency).
Each is chosen so that a plausible slip in the oracle (dropped scale, wrong
group mapping, off-by-one causal bound, transposed page layout, wrong row of a
packed query) fails at least one of them.
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle
from tests.refs import bf16_bits, bits_f64, dense_rows, place, randn_bits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _sdpa(q, k, v, mask, scale):
    """torch fp64 SDPA. q [Hq][Tq][D], k/v [Hkv][L][D], mask bool [Tq][L]."""
    return torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None], torch.from_numpy(k)[None], torch.from_numpy(v)[None],
        attn_mask=torch.from_numpy(mask)[None, None], scale=scale, enable_gqa=True)[0].numpy()


def _rand_rows(rng, lens, Hkv, D):
    ks = [randn_bits(rng, (Hkv, L, D)) for L in lens]
    vs = [randn_bits(rng, (Hkv, L, D)) for L in lens]
    return ks, vs


# ---------------------------------------------------------------- fixtures

def _read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def test_golden_page_layout():
    """Hand-derived flat offsets of a tiny page write (tests/golden/page_layout_tiny.txt)."""
    Hkv, P, D = 2, 2, 2
    t, g, d = np.meshgrid(np.arange(3), np.arange(Hkv), np.arange(D), indexing="ij")
    k_new = (100 + 4 * t + 2 * g + d).astype(np.uint16)
    v_new = (200 + 4 * t + 2 * g + d).astype(np.uint16)
    kp = np.zeros((4, Hkv, P, D), np.uint16)
    vp = np.zeros((4, Hkv, D, P), np.uint16)
    bt = np.array([[3, 1]], np.int32)
    kp2, vp2 = oracle.page_write(k_new, v_new, [0, 3], [0], bt, kp, vp)
    want_k = np.zeros(32, np.uint16)
    want_v = np.zeros(32, np.uint16)
    for pool, idx, val in _read_golden("page_layout_tiny.txt"):
        (want_k if pool == "K" else want_v)[int(idx)] = int(val)
    np.testing.assert_array_equal(kp2.reshape(-1), want_k)
    np.testing.assert_array_equal(vp2.reshape(-1), want_v)
    # the gather of the written positions returns exactly the new tokens
    ko, vo = oracle.page_gather(kp2, vp2, bt, [3], [0, 3])
    np.testing.assert_array_equal(ko, k_new)
    np.testing.assert_array_equal(vo, v_new)


def test_golden_two_keys():
    """Hand-worked two-key example (tests/golden/attn_two_keys.txt)."""
    want = {k: float(v) for k, v in _read_golden("attn_two_keys.txt")}
    q = bf16_bits([[[1.0, 0.0]]])
    kp = np.zeros((1, 1, 2, 2), np.uint16)
    vp = np.zeros((1, 1, 2, 2), np.uint16)
    kp[0, 0, 0] = bf16_bits([0.0, 0.0])
    kp[0, 0, 1] = bf16_bits([2.0, 0.0])
    vp[0, 0, :, 0] = bf16_bits([1.0, 0.0])   # v0 (V pages are dim-major)
    vp[0, 0, :, 1] = bf16_bits([0.0, 1.0])   # v1
    out, lse = oracle.decode(q, kp, vp, np.zeros((1, 1), np.int32), [2], 1.0)
    assert abs(out[0, 0, 0] - want["out0"]) < 1e-15
    assert abs(out[0, 0, 1] - want["out1"]) < 1e-15
    assert abs(lse[0, 0] - want["lse"]) < 1e-15


# ------------------------------------------------------- library routine

@pytest.mark.parametrize("Hq,Hkv,P,D", [(2, 1, 16, 128), (4, 2, 16, 128), (8, 2, 16, 128),
                                        (8, 2, 4, 8), (6, 3, 2, 4)])
def test_decode_matches_torch_sdpa(Hq, Hkv, P, D):
    rng = np.random.default_rng(Hq * 100 + Hkv * 10 + P)
    lens = [1, 17, 40, 16, 33]
    ks, vs = _rand_rows(rng, lens, Hkv, D)
    kp, vp, bt = place(ks, vs, 0, Hkv, P, D, rng)
    q = randn_bits(rng, (len(lens), Hq, D))
    scale = 1.0 / math.sqrt(D)
    out, lse = oracle.decode(q, kp, vp, bt, lens, scale)
    for b, L in enumerate(lens):
        ref = _sdpa(bits_f64(q[b])[:, None, :], bits_f64(ks[b]), bits_f64(vs[b]),
                    np.ones((1, L), bool), scale)[:, 0, :]
        np.testing.assert_allclose(out[b], ref, rtol=1e-12, atol=1e-13)
        # lse against a log-sum-exp of the library's own matmul scores
        kk = torch.from_numpy(bits_f64(ks[b])).repeat_interleave(Hq // Hkv, 0)
        s = torch.einsum("hd,hjd->hj", torch.from_numpy(bits_f64(q[b])), kk) * scale
        np.testing.assert_allclose(lse[b], torch.logsumexp(s, -1).numpy(), rtol=1e-13)


@pytest.mark.parametrize("Hq,Hkv,P,D", [(2, 1, 16, 128), (8, 2, 16, 128), (4, 4, 4, 8)])
def test_append_matches_torch_sdpa(Hq, Hkv, P, D):
    rng = np.random.default_rng(7 + Hq + P)
    ctx = [0, 1, 15, 16, 17]
    T = [5, 20, 1, 16, 3]
    lens = [c + t for c, t in zip(ctx, T)]
    ks, vs = _rand_rows(rng, lens, Hkv, D)
    kp, vp, bt = place(ks, vs, 0, Hkv, P, D, rng)
    cu = np.concatenate([[0], np.cumsum(T)]).astype(np.int32)
    q = randn_bits(rng, (int(cu[-1]), Hq, D))
    scale = 1.0 / math.sqrt(D)
    out, lse = oracle.append(q, cu, ctx, kp, vp, bt, scale)
    for b in range(len(ctx)):
        qb = bits_f64(q[cu[b]:cu[b + 1]]).transpose(1, 0, 2)          # [Hq][T][D]
        i = np.arange(T[b])[:, None]
        j = np.arange(lens[b])[None, :]
        mask = j <= ctx[b] + i                                         # bottom-right causal
        ref = _sdpa(qb, bits_f64(ks[b]), bits_f64(vs[b]), mask, scale).transpose(1, 0, 2)
        np.testing.assert_allclose(out[cu[b]:cu[b + 1]], ref, rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------- brute force

def test_decode_dense_bruteforce_reads_pages_by_subscript():
    """Dense numpy attention over K/V read back through block-table subscripts."""
    rng = np.random.default_rng(11)
    Hq, Hkv, P, D = 8, 2, 16, 128
    lens = [3, 40, 32, 1]
    ks, vs = _rand_rows(rng, lens, Hkv, D)
    kp, vp, bt = place(ks, vs, 64, Hkv, P, D, rng)
    q = randn_bits(rng, (len(lens), Hq, D))
    scale = 1.0 / math.sqrt(D)
    out, _ = oracle.decode(q, kp, vp, bt, lens, scale)
    kd, vd = dense_rows(kp, vp, bt, lens)
    G = Hq // Hkv
    for b in range(len(lens)):
        for h in range(Hq):
            s = bits_f64(kd[b][h // G]) @ bits_f64(q[b, h]) * scale
            w = np.exp(s - s.max())
            ref = (w[:, None] * bits_f64(vd[b][h // G])).sum(0) / w.sum()
            np.testing.assert_allclose(out[b, h], ref, rtol=1e-12, atol=1e-14)


# ------------------------------------------------------------ closed forms

def test_one_key_returns_that_value_row_exactly():
    rng = np.random.default_rng(3)
    Hq, Hkv, P, D = 4, 2, 16, 128
    ks, vs = _rand_rows(rng, [1, 1], Hkv, D)
    kp, vp, bt = place(ks, vs, 0, Hkv, P, D, rng)
    q = randn_bits(rng, (2, Hq, D))
    out, lse = oracle.decode(q, kp, vp, bt, [1, 1], 0.088)
    for b in range(2):
        for h in range(Hq):
            np.testing.assert_array_equal(out[b, h], bits_f64(vs[b][h // 2, 0]))
            s = 0.088 * float(np.dot(bits_f64(q[b, h]), bits_f64(ks[b][h // 2, 0])))
            assert abs(lse[b, h] - s) <= 1e-14 * max(1.0, abs(s))
    # append with no cached context and a one-token chunk is the same case
    out_a, _ = oracle.append(q[:1], [0, 1], [0], kp, vp, bt[:1], 0.088)
    np.testing.assert_array_equal(out_a[0], out[0])


@pytest.mark.parametrize("scale", [0.0, 1.0 / math.sqrt(128)])
def test_identical_keys_give_mean_of_values(scale):
    rng = np.random.default_rng(5)
    Hq, Hkv, P, D, L = 4, 1, 16, 128, 37
    k1 = randn_bits(rng, (Hkv, 1, D))
    ks = [np.repeat(k1, L, axis=1)] if scale else [randn_bits(rng, (Hkv, L, D))]
    vs = [randn_bits(rng, (Hkv, L, D))]
    kp, vp, bt = place(ks, vs, 0, Hkv, P, D, rng)
    q = randn_bits(rng, (1, Hq, D))
    out, lse = oracle.decode(q, kp, vp, bt, [L], scale)
    mean = bits_f64(vs[0][0]).mean(0)
    for h in range(Hq):
        np.testing.assert_allclose(out[0, h], mean, rtol=1e-13, atol=1e-15)
        s = scale * float(np.dot(bits_f64(q[0, h]), bits_f64(ks[0][0, 0])))
        assert abs(lse[0, h] - (s + math.log(L))) < 1e-12


def test_two_keys_sigmoid_closed_form():
    rng = np.random.default_rng(9)
    Hq, Hkv, P, D = 8, 2, 16, 128
    ks, vs = _rand_rows(rng, [2], Hkv, D)
    kp, vp, bt = place(ks, vs, 0, Hkv, P, D, rng)
    q = randn_bits(rng, (1, Hq, D))
    scale = 0.3
    out, lse = oracle.decode(q, kp, vp, bt, [2], scale)
    for h in range(Hq):
        g = h // 4
        s0 = scale * np.dot(bits_f64(q[0, h]), bits_f64(ks[0][g, 0]))
        s1 = scale * np.dot(bits_f64(q[0, h]), bits_f64(ks[0][g, 1]))
        sig = lambda x: 1.0 / (1.0 + math.exp(-x))
        ref = sig(s0 - s1) * bits_f64(vs[0][g, 0]) + sig(s1 - s0) * bits_f64(vs[0][g, 1])
        np.testing.assert_allclose(out[0, h], ref, rtol=1e-12, atol=1e-14)
        assert abs(lse[0, h] - (max(s0, s1) + math.log1p(math.exp(-abs(s0 - s1))))) < 1e-12


def test_empty_row_gives_zero_and_minus_inf():
    rng = np.random.default_rng(1)
    ks, vs = _rand_rows(rng, [4, 1], 1, 128)
    kp, vp, bt = place(ks, vs, 0, 1, 16, 128, rng)
    q = randn_bits(rng, (2, 2, 128))
    out, lse = oracle.decode(q, kp, vp, bt, [0, 1], 0.1)
    assert np.all(out[0] == 0.0) and np.all(np.isneginf(lse[0]))
    assert np.all(np.isfinite(out[1]))


# -------------------------------------------------------------- invariants

def test_page_permutation_invariance_is_exact():
    rng = np.random.default_rng(21)
    Hq, Hkv, P, D = 8, 2, 16, 128
    lens = [50, 7, 64]
    ks, vs = _rand_rows(rng, lens, Hkv, D)
    q = randn_bits(rng, (3, Hq, D))
    kp1, vp1, bt1 = place(ks, vs, 40, Hkv, P, D, np.random.default_rng(1))
    kp2, vp2, bt2 = place(ks, vs, 40, Hkv, P, D, np.random.default_rng(2))
    assert not np.array_equal(bt1, bt2)
    o1, l1 = oracle.decode(q, kp1, vp1, bt1, lens, 0.09)
    o2, l2 = oracle.decode(q, kp2, vp2, bt2, lens, 0.09)
    np.testing.assert_array_equal(o1, o2)
    np.testing.assert_array_equal(l1, l2)


def test_causal_mask_respected_and_prefix_consistent():
    rng = np.random.default_rng(31)
    Hq, Hkv, P, D = 4, 2, 16, 128
    ctx, T = 19, 14
    ks, vs = _rand_rows(rng, [ctx + T], Hkv, D)
    kp, vp, bt = place(ks, vs, 0, Hkv, P, D, rng)
    q = randn_bits(rng, (T, Hq, D))
    out, _ = oracle.append(q, [0, T], [ctx], kp, vp, bt, 0.1)
    for i in [0, 5, T - 2]:
        # perturb every key/value after position ctx + i
        ks2 = [ks[0].copy()]
        vs2 = [vs[0].copy()]
        ks2[0][:, ctx + i + 1:, :] = randn_bits(rng, ks2[0][:, ctx + i + 1:, :].shape)
        vs2[0][:, ctx + i + 1:, :] = randn_bits(rng, vs2[0][:, ctx + i + 1:, :].shape)
        kp2, vp2, bt2 = place(ks2, vs2, 0, Hkv, P, D, np.random.default_rng(0))
        out2, _ = oracle.append(q, [0, T], [ctx], kp2, vp2, bt2, 0.1)
        np.testing.assert_array_equal(out2[i], out[i])
        assert not np.array_equal(out2[T - 1], out[T - 1])
        # a shorter chunk ending at query i gives the same row i
        out3, _ = oracle.append(q[:i + 1], [0, i + 1], [ctx], kp, vp, bt, 0.1)
        np.testing.assert_array_equal(out3[i], out[i])


def test_append_one_token_equals_decode():
    rng = np.random.default_rng(41)
    Hq, Hkv, P, D = 8, 2, 16, 128
    ctx = [0, 16, 31]
    ks, vs = _rand_rows(rng, [c + 1 for c in ctx], Hkv, D)
    kp, vp, bt = place(ks, vs, 0, Hkv, P, D, rng)
    q = randn_bits(rng, (3, Hq, D))
    oa, la = oracle.append(q, [0, 1, 2, 3], ctx, kp, vp, bt, 0.1)
    od, ld = oracle.decode(q, kp, vp, bt, [c + 1 for c in ctx], 0.1)
    np.testing.assert_array_equal(oa, od)
    np.testing.assert_array_equal(la, ld)


def test_key_shift_and_value_affinity():
    rng = np.random.default_rng(51)
    Hq, Hkv, P, D, L = 4, 2, 16, 128, 45
    # small-integer keys and values so that +c, *2 and +1 stay exact in bf16
    k = bf16_bits(rng.integers(-4, 5, (Hkv, L, D)))
    v = bf16_bits(rng.integers(-8, 9, (Hkv, L, D)))
    c = rng.integers(-2, 3, (Hkv, 1, D))
    k_shift = bf16_bits(bits_f64(k) + c)
    v_aff = bf16_bits(2.0 * bits_f64(v) + 1.0)
    q = randn_bits(rng, (1, Hq, D))
    run = lambda kk, vv: oracle.decode(q, *place([kk], [vv], 0, Hkv, P, D,
                                                 np.random.default_rng(0)), [L], 0.05)
    o, _ = run(k, v)
    o_shift, _ = run(k_shift, v)
    o_aff, _ = run(k, v_aff)
    np.testing.assert_allclose(o_shift, o, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(o_aff, 2.0 * o + 1.0, rtol=1e-12, atol=1e-12)


def test_group_consistency():
    """Heads of one group with equal queries give equal outputs; other groups differ."""
    rng = np.random.default_rng(61)
    Hq, Hkv, P, D = 8, 2, 16, 128
    ks, vs = _rand_rows(rng, [30], Hkv, D)
    kp, vp, bt = place(ks, vs, 0, Hkv, P, D, rng)
    q1 = randn_bits(rng, (D,))
    q = np.broadcast_to(q1, (1, Hq, D)).copy()
    out, _ = oracle.decode(q, kp, vp, bt, [30], 0.1)
    for h in range(1, 4):
        np.testing.assert_array_equal(out[0, h], out[0, 0])
        np.testing.assert_array_equal(out[0, 4 + h], out[0, 4])
    assert not np.array_equal(out[0, 0], out[0, 4])


# ------------------------------------------------------ page write / gather

def test_page_write_then_gather_roundtrip_and_untouched():
    rng = np.random.default_rng(71)
    Hkv, P, D = 2, 16, 128
    old = [37, 0, 16, 5]
    new = [1, 20, 33, 0]
    total = [o + n for o, n in zip(old, new)]
    ks, vs = _rand_rows(rng, total, Hkv, D)
    kp, vp, bt = place(ks, vs, 0, Hkv, P, D, rng)
    cu = np.concatenate([[0], np.cumsum(new)]).astype(np.int32)
    k_new = randn_bits(rng, (int(cu[-1]), Hkv, D))
    v_new = randn_bits(rng, (int(cu[-1]), Hkv, D))
    kp2, vp2 = oracle.page_write(k_new, v_new, cu, old, bt, kp, vp)
    # expected pools built with numpy subscripts
    kx, vx = kp.copy(), vp.copy()
    for b in range(4):
        for t in range(new[b]):
            pos = old[b] + t
            kx[bt[b, pos // P], :, pos % P, :] = k_new[cu[b] + t]
            vx[bt[b, pos // P], :, :, pos % P] = v_new[cu[b] + t]
    np.testing.assert_array_equal(kp2, kx)
    np.testing.assert_array_equal(vp2, vx)
    assert np.sum(kp2 != kp) > 0
    # gather of the full rows: old prefix unchanged, new tokens in place
    cu_out = np.concatenate([[0], np.cumsum(total)]).astype(np.int32)
    ko, vo = oracle.page_gather(kp2, vp2, bt, total, cu_out)
    for b in range(4):
        kr = ko[cu_out[b]:cu_out[b + 1]].transpose(1, 0, 2)
        vr = vo[cu_out[b]:cu_out[b + 1]].transpose(1, 0, 2)
        np.testing.assert_array_equal(kr[:, :old[b]], ks[b][:, :old[b]])
        np.testing.assert_array_equal(vr[:, :old[b]], vs[b][:, :old[b]])
        np.testing.assert_array_equal(kr[:, old[b]:].transpose(1, 0, 2), k_new[cu[b]:cu[b + 1]])
        np.testing.assert_array_equal(vr[:, old[b]:].transpose(1, 0, 2), v_new[cu[b]:cu[b + 1]])


def test_gather_matches_subscript_reading():
    rng = np.random.default_rng(81)
    Hkv, P, D = 3, 4, 8
    lens = [9, 1, 12]
    ks, vs = _rand_rows(rng, lens, Hkv, D)
    kp, vp, bt = place(ks, vs, 0, Hkv, P, D, rng)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    ko, vo = oracle.page_gather(kp, vp, bt, lens, cu)
    kd, vd = dense_rows(kp, vp, bt, lens)
    for b in range(3):
        np.testing.assert_array_equal(ko[cu[b]:cu[b + 1]], kd[b].transpose(1, 0, 2))
        np.testing.assert_array_equal(vo[cu[b]:cu[b + 1]], vd[b].transpose(1, 0, 2))
        np.testing.assert_array_equal(kd[b], ks[b])


# ----------------------------------------------------------------------------- token log-probs

def _golden(name):
    vals = {}
    for line in open(os.path.join(GOLDEN, name)):
        if line.strip() and not line.startswith("#"):
            k, v = line.split()
            vals[k] = float(v)
    return vals


def test_logprob_matches_library_log_softmax():
    """numpy fp64 matmul + scipy's log_softmax (an independent implementation)."""
    from scipy.special import log_softmax
    rng = np.random.default_rng(71)
    N, V, D = 5, 37, 48
    h, W = randn_bits(rng, (N, D)), randn_bits(rng, (V, D))
    t = np.array([0, 36, 5, 17, 5], np.int32)
    for scale in (1.0, 0.7):
        z = scale * (bits_f64(h) @ bits_f64(W).T)          # [N][V]
        ref = log_softmax(z, axis=1)
        logp, lse = oracle.token_logprob(h, W, t, scale)
        np.testing.assert_allclose(logp, ref[np.arange(N), t], rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse, z[np.arange(N), t] - ref[np.arange(N), t], rtol=1e-13)


def test_logprob_golden_three_tokens():
    g = _golden("logprob_three_tokens.txt")
    h = bf16_bits([[1.0, 0.0]] * 3)
    W = bf16_bits([[0.0, 0.0], [1.0, 0.0], [2.0, 0.0]])
    logp, lse = oracle.token_logprob(h, W, [0, 1, 2])
    for i in range(3):
        assert abs(logp[i] - g[f"logp{i}"]) < 1e-14
        assert abs(lse[i] - g["lse"]) < 1e-14


def test_logprob_closed_forms():
    rng = np.random.default_rng(72)
    V, D = 29, 32
    W = randn_bits(rng, (V, D))
    # zero hidden state: uniform distribution
    logp, lse = oracle.token_logprob(np.zeros((2, D), np.uint16), W, [0, 28])
    np.testing.assert_allclose(logp, -math.log(V), rtol=0, atol=1e-15)
    np.testing.assert_allclose(lse, math.log(V), rtol=0, atol=1e-15)
    # out-of-range targets have no log-probability; lse is unaffected
    h = randn_bits(rng, (3, D))
    logp, lse = oracle.token_logprob(h, W, [-1, V, 3])
    assert np.isnan(logp[0]) and np.isnan(logp[1]) and np.isfinite(logp[2])
    assert np.all(np.isfinite(lse))
    # logits of 1000 and 996 (exact in bf16): exp overflows fp64 unless the
    # maximum is taken out first; lse = 1000 + ln(1 + e^-4)
    h = bf16_bits([[1.0, 0.0]] * 2)
    W = bf16_bits([[1000.0, 0.0], [996.0, 0.0]])
    logp, lse = oracle.token_logprob(h, W, [0, 1])
    np.testing.assert_allclose(lse, 1000.0 + math.log1p(math.exp(-4.0)), rtol=0, atol=1e-12)
    np.testing.assert_allclose(logp, [-math.log1p(math.exp(-4.0)), -4.0 - math.log1p(math.exp(-4.0))],
                               rtol=0, atol=1e-12)


def test_logprob_normalised_and_shift_invariant():
    rng = np.random.default_rng(73)
    V, D = 23, 16
    # small integers: every product and sum below is exact in bf16 and fp64
    h = bf16_bits(rng.integers(-2, 3, size=(1, D)))
    W = bf16_bits(rng.integers(-2, 3, size=(V, D)))
    all_t = np.arange(V, dtype=np.int32)
    logp, _ = oracle.token_logprob(np.repeat(h, V, 0), W, all_t)
    assert abs(math.fsum(np.exp(logp)) - 1.0) < 1e-14
    # adding one vector w0 to every row shifts all logits by <h, w0>: no change
    w0 = rng.integers(-2, 3, size=D)
    W2 = bf16_bits(bits_f64(W) + w0)
    logp2, lse2 = oracle.token_logprob(np.repeat(h, V, 0), W2, all_t)
    np.testing.assert_allclose(logp2, logp, rtol=0, atol=1e-13)
    shift = float(bits_f64(h)[0] @ w0)
    _, lse1 = oracle.token_logprob(np.repeat(h, V, 0), W, all_t)
    np.testing.assert_allclose(lse2, lse1 + shift, rtol=0, atol=1e-12)


# ----------------------------------------------------------------------------- fp8 pools

def test_e4m3_decode_matches_torch_for_every_code():
    """The E4M3 value table against torch's float8_e4m3fn (a library routine)."""
    c = np.arange(256, dtype=np.uint8)
    mine = oracle.e4m3_decode(c)
    ref = torch.from_numpy(c).view(torch.float8_e4m3fn).double().numpy()
    assert np.array_equal(np.isnan(mine), np.isnan(ref))
    assert np.isnan(mine[[0x7F, 0xFF]]).all() and np.isnan(mine).sum() == 2
    ok = ~np.isnan(ref)
    np.testing.assert_array_equal(mine[ok], ref[ok])
    assert mine[0x7E] == 448.0 and mine[0x01] == 2.0 ** -9 and mine[0x38] == 1.0


def test_e4m3_encode_matches_torch_in_range():
    """Round to nearest (ties to even) against torch for every finite bf16 value within
    +-448 and for random fp32 values across the subnormal and normal ranges."""
    b = np.arange(1 << 16, dtype=np.uint32)
    f = (b << 16).view(np.float32)
    f = f[np.isfinite(f) & (np.abs(f) <= 448)]
    rng = np.random.default_rng(3)
    r = (rng.standard_normal(100000) * 2.0 ** rng.integers(-14, 9, 100000)).astype(np.float32)
    x = np.concatenate([f, r[np.abs(r) <= 448]])
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    np.testing.assert_array_equal(oracle.e4m3_encode(x), ref)


def test_e4m3_encode_closed_forms():
    cases = [
        (1.0, 0x38), (-1.0, 0xB8), (448.0, 0x7E), (-448.0, 0xFE),
        (1.0625, 0x38),   # halfway between 1 and 1.125: the even code
        (1.1875, 0x3A),   # halfway between 1.125 and 1.25: the even code
        (2.0 ** -9, 0x01),   # smallest subnormal
        (2.0 ** -10, 0x00),   # half of it: tie to the even code 0
        (3 * 2.0 ** -10, 0x02),   # halfway between 2^-9 and 2^-8: even
        (-0.0, 0x80), (0.0, 0x00),
        (464.0, 0x7E), (1e6, 0x7E), (-1e6, 0xFE),   # saturation
        (float("inf"), 0x7E), (float("-inf"), 0xFE),
        (float("nan"), 0x7F),
    ]
    x = np.array([c[0] for c in cases], np.float64)
    np.testing.assert_array_equal(oracle.e4m3_encode(x), np.array([c[1] for c in cases], np.uint8))
    # decode(encode(v)) == v for every finite code's value
    c = np.array([i for i in range(256) if i not in (0x7F, 0xFF)], np.uint8)
    np.testing.assert_array_equal(oracle.e4m3_encode(oracle.e4m3_decode(c)), c)


def _fp8_pools(rng, lens, Hkv, P, D):
    """Paged fp8 pools holding random finite codes (the layout of place())."""
    ks = [rng.integers(0, 0x7F, (Hkv, L, D)) | (rng.integers(0, 2, (Hkv, L, D)) << 7)
          for L in lens]
    vs = [rng.integers(0, 0x7F, (Hkv, L, D)) | (rng.integers(0, 2, (Hkv, L, D)) << 7)
          for L in lens]
    kp, vp, bt = place([k.astype(np.uint16) for k in ks], [v.astype(np.uint16) for v in vs], 0,
                       Hkv, P, D, rng, fill=0)
    return kp.astype(np.uint8), vp.astype(np.uint8), bt


def test_fp8_page_write_quantizes_and_gathers_codes():
    rng = np.random.default_rng(91)
    Hkv, P, D = 2, 16, 128
    old, new = [37, 0, 16, 5], [1, 20, 33, 0]
    total = [o + n for o, n in zip(old, new)]
    kp, vp, bt = _fp8_pools(rng, total, Hkv, P, D)
    cu = np.concatenate([[0], np.cumsum(new)]).astype(np.int32)
    k_new = randn_bits(rng, (int(cu[-1]), Hkv, D))
    v_new = bf16_bits(rng.standard_normal((int(cu[-1]), Hkv, D)) * 300.0)   # some saturate
    ks, vs = 0.05, 0.7
    kp2, vp2 = oracle.page_write_fp8(k_new, v_new, cu, old, bt, kp, vp, ks, vs)
    kq, vq = oracle.quantize(k_new, ks), oracle.quantize(v_new, vs)
    kx, vx = kp.copy(), vp.copy()
    for b in range(4):
        for t in range(new[b]):
            pos = old[b] + t
            kx[bt[b, pos // P], :, pos % P, :] = kq[cu[b] + t]
            vx[bt[b, pos // P], :, :, pos % P] = vq[cu[b] + t]
    np.testing.assert_array_equal(kp2, kx)
    np.testing.assert_array_equal(vp2, vx)
    assert (vq == 0x7E).any() or (vq == 0xFE).any()
    # the stored value is within half a quantum of x / scale (or saturated)
    xk = bits_f64(k_new) / np.float32(ks)
    dk = oracle.e4m3_decode(kq)
    assert np.all(np.abs(dk - xk) <= np.maximum(np.abs(xk) * 2.0 ** -4, 2.0 ** -10) + 1e-12)
    cu_out = np.concatenate([[0], np.cumsum(total)]).astype(np.int32)
    ko, vo = oracle.page_gather_u8(kp2, vp2, bt, total, cu_out)
    kd, vd = dense_rows(kp2, vp2, bt, total)
    for b in range(4):
        np.testing.assert_array_equal(ko[cu_out[b]:cu_out[b + 1]], kd[b].transpose(1, 0, 2))
        np.testing.assert_array_equal(vo[cu_out[b]:cu_out[b + 1]], vd[b].transpose(1, 0, 2))


@pytest.mark.parametrize("ks,vs", [(2.0 ** -3, 2.0 ** 2), (1.0, 2.0 ** -5)])
def test_fp8_attention_equals_bf16_oracle_on_exact_values(ks, vs):
    """With power-of-two scales every dequantized value is exactly a bf16 value, so
    attention over the fp8 pools must equal the (pinned) bf16 oracle bitwise."""
    rng = np.random.default_rng(int(ks * 64 + vs))
    Hq, Hkv, P, D = 8, 2, 16, 128
    lens = [1, 17, 40, 0, 33]
    kp, vp, bt = _fp8_pools(rng, lens, Hkv, P, D)
    kb = bf16_bits(oracle.e4m3_decode(kp) * ks)
    vb = bf16_bits(oracle.e4m3_decode(vp) * vs)
    np.testing.assert_array_equal(bits_f64(kb), oracle.e4m3_decode(kp) * ks)
    q = randn_bits(rng, (len(lens), Hq, D))
    a, la = oracle.decode_fp8(q, kp, vp, ks, vs, bt, lens, 0.03)
    b, lb = oracle.decode(q, kb, vb, bt, lens, 0.03)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(la, lb)
    T = [1, 5, 7, 0, 9]
    T = [min(t, L) for t, L in zip(T, lens)]
    ctx = [L - t for L, t in zip(lens, T)]
    cu = np.concatenate([[0], np.cumsum(T)]).astype(np.int32)
    qa = randn_bits(rng, (int(cu[-1]), Hq, D))
    a, la = oracle.append_fp8(qa, cu, ctx, kp, vp, ks, vs, bt, 0.03)
    b, lb = oracle.append(qa, cu, ctx, kb, vb, bt, 0.03)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(la, lb)


def test_fp8_scale_laws():
    """k_scale multiplies every score (it folds into the softmax scale); v_scale
    multiplies the output and leaves lse unchanged."""
    rng = np.random.default_rng(5)
    Hq, Hkv, P, D = 4, 1, 16, 128
    lens = [3, 50]
    kp, vp, bt = _fp8_pools(rng, lens, Hkv, P, D)
    q = randn_bits(rng, (2, Hq, D))
    a, la = oracle.decode_fp8(q, kp, vp, 0.3, 1.7, bt, lens, 0.01)
    b, lb = oracle.decode_fp8(q, kp, vp, 1.0, 1.0, bt, lens, 0.003)
    np.testing.assert_allclose(a, 1.7 * b, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(la, lb, rtol=1e-12, atol=1e-12)


def _rope_table(theta, positions):
    """cos | sin of the angles p * theta^(-2i/128), i < 64, for the given positions
    (fp64 math, stored fp32): the table a caller builds for its model."""
    inv = float(theta) ** (-2.0 * np.arange(64) / 128.0)
    ang = np.asarray(positions, np.float64)[:, None] * inv[None, :]
    return np.concatenate([np.cos(ang), np.sin(ang)], axis=1).astype(np.float32)


def test_rope_identity_at_angle_zero():
    """Position 0 (cos 1, sin 0) leaves every row bit for bit."""
    rng = np.random.default_rng(21)
    x = randn_bits(rng, (7, 3, 128))
    table = _rope_table(1e6, np.arange(8))
    np.testing.assert_array_equal(oracle.rope(x, np.zeros(7, np.int32), table), x)


def test_rope_is_the_complex_rotation_of_dim_pairs():
    """Dims i and i + 64 form the complex number x_i + j x_{i+64}, multiplied by
    e^{j angle_i}: the rotation computed as a complex product in fp64 agrees with
    the oracle to within one bf16 step everywhere and exactly almost everywhere
    (the oracle rounds its products to fp32 first). A swapped pairing
    (2i, 2i+1) or a flipped sign fails."""
    rng = np.random.default_rng(22)
    N, H = 64, 4
    x = randn_bits(rng, (N, H, 128))
    table = _rope_table(1e4, np.arange(5000))
    pos = rng.integers(0, 5000, N).astype(np.int32)
    y = bits_f64(oracle.rope(x, pos, table))
    xf = bits_f64(x)
    c = table[pos, :64].astype(np.float64)[:, None, :]
    s = table[pos, 64:].astype(np.float64)[:, None, :]
    z = (xf[..., :64] + 1j * xf[..., 64:]) * (c + 1j * s)
    ref = np.concatenate([z.real, z.imag], axis=-1)
    ulp = np.abs(bits_f64(bf16_bits(ref))) * 2.0 ** -7 + 1e-30
    err = np.abs(y - ref)
    assert np.all(err <= ulp + 1e-12)
    assert np.mean(y == bits_f64(bf16_bits(ref))) > 0.99


def test_rope_bits_follow_the_stated_fp32_rounding():
    """The rotation's rounding, restated independently: numpy float32 products
    x_i c_i, x_{i+64} s_i, x_{i+64} c_i, x_i s_i (each rounded to fp32), numpy
    float32 difference and sum (rounded to fp32), then torch's round-to-nearest-
    even conversion to bf16. The oracle must equal it on every element, bit for
    bit. On the same inputs the two plausible other readings (the rotation in
    fp64 rounded once to bf16; fused multiply-adds, x_i c_i - x_{i+64} s_i with
    one rounding) differ from it on some elements, so the pin tells them apart."""
    rng = np.random.default_rng(25)
    N, H = 512, 4
    x = randn_bits(rng, (N, H, 128))
    # a few large and tiny magnitudes, and exact zeros, among the normal values
    x[0, 0, :8] = bf16_bits(np.array([3e38, -3e38, 1e-38, -1e-38, 0.0, -0.0, 65504.0, 1e-5]))
    table = _rope_table(1e6, np.arange(40000))
    pos = rng.integers(0, 40000, N).astype(np.int32)
    got = oracle.rope(x, pos, table)

    xf = bits_f64(x).astype(np.float32)
    lo, hi = xf[..., :64], xf[..., 64:]
    c = table[pos, None, :64]
    s = table[pos, None, 64:]
    with np.errstate(over="ignore", invalid="ignore"):
        y_lo = np.float32(lo * c) - np.float32(hi * s)
        y_hi = np.float32(hi * c) + np.float32(lo * s)
    y32 = np.concatenate([y_lo, y_hi], axis=-1)
    assert y32.dtype == np.float32
    want = torch.from_numpy(y32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(got, want)

    # the alternative readings differ from this one somewhere
    lo64, hi64 = lo.astype(np.float64), hi.astype(np.float64)
    c64, s64 = c.astype(np.float64), s.astype(np.float64)
    with np.errstate(over="ignore", invalid="ignore"):
        f64 = np.concatenate([lo64 * c64 - hi64 * s64, hi64 * c64 + lo64 * s64], axis=-1)
        fma = np.concatenate([(lo64 * c64 - np.float32(hi * s)).astype(np.float32),
                              (hi64 * c64 + np.float32(lo * s)).astype(np.float32)], axis=-1)
    once = torch.from_numpy(f64.astype(np.float32)).to(torch.bfloat16)
    fused = torch.from_numpy(fma).to(torch.bfloat16)
    for alt in (once, fused):
        alt_bits = alt.view(torch.int16).numpy().view(np.uint16)
        assert np.any(alt_bits != want)


def test_rope_scores_depend_on_relative_position_only():
    """<rot(q, p1), rot(k, p2)> is a function of p1 - p2: shifting both
    positions by d changes it only by bf16 rounding."""
    rng = np.random.default_rng(23)
    q = randn_bits(rng, (1, 1, 128))
    k = randn_bits(rng, (1, 1, 128))
    table = _rope_table(1e6, np.arange(40000))
    for p1, p2, d in [(5, 3, 1000), (30000, 17, 7777), (100, 9000, 20000)]:
        a = np.sum(bits_f64(oracle.rope(q, [p1], table)) * bits_f64(oracle.rope(k, [p2], table)))
        b = np.sum(bits_f64(oracle.rope(q, [p1 + d], table)) *
                   bits_f64(oracle.rope(k, [p2 + d], table)))
        assert abs(a - b) < 0.1, (p1, p2, d, a, b)
    # and it does change with the relative position
    a = np.sum(bits_f64(oracle.rope(q, [5], table)) * bits_f64(oracle.rope(k, [3], table)))
    b = np.sum(bits_f64(oracle.rope(q, [5], table)) * bits_f64(oracle.rope(k, [30003], table)))
    assert abs(a - b) > 0.5


def test_rope_inverse_rotation_and_pair_norms():
    """Rotating by an angle and then by its negative returns the row (to bf16
    rounding), and each pair's norm is kept."""
    rng = np.random.default_rng(24)
    x = randn_bits(rng, (16, 2, 128))
    p = 12345.0
    table = _rope_table(1e4, [0.0, p, -p])
    y = oracle.rope(x, np.ones(16, np.int32), table)
    back = oracle.rope(y, np.full(16, 2, np.int32), table)
    np.testing.assert_allclose(bits_f64(back), bits_f64(x), rtol=2 ** -6, atol=2 ** -7)
    xf, yf = bits_f64(x), bits_f64(y)
    n0 = xf[..., :64] ** 2 + xf[..., 64:] ** 2
    n1 = yf[..., :64] ** 2 + yf[..., 64:] ** 2
    np.testing.assert_allclose(n1, n0, rtol=2 ** -6, atol=1e-3)
