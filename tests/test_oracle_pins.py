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
