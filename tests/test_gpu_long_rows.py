"""Very long rows against the fp64 oracle (through the C ABI).

A decode row of 1,048,576 keys (65,536 pages, 2 GiB of bf16 K per pool) beside
rows of 17 and 4,101 keys: the longest row takes 256 splits of 4,096 keys, so
the combine merges far more partials than in any benchmark workload, and the
short rows leave most of their splits empty. An append chunk of 300 queries
after a 262,144-token context, beside a chunk with no context, checked on
sampled queries through the identity append query i == decode of ctx + i + 1
keys. The no-allocation decode takes the million-key batch too (its plan fits
the static scratch array) and must equal the ordinary call bit for bit.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2603_18815_amd as ra
import synth
from tests.gpu_util import (APPEND_LSE_ATOL, DECODE_LSE_ATOL, assert_attn_close, bits,
                            compact_rows)

pytestmark = pytest.mark.gpu
SCALE = 1.0 / math.sqrt(128)


def i32(x, dev):
    return torch.as_tensor(np.ascontiguousarray(np.asarray(x, np.int32)), device=dev)


def say(msg):
    print(f"[gpu-test] {msg}", flush=True)


def pools(seed, lens, Hkv, dev):
    rng = np.random.default_rng(seed)
    lay = synth.make_layout(rng, lens)
    gen = synth.value_generator(seed, dev)
    k = synth.randn_bf16((lay.num_pages, Hkv, 16, 128), gen, dev)
    v = synth.randn_bf16((lay.num_pages, Hkv, 128, 16), gen, dev)
    return lay, k, v, gen


def test_decode_million_key_row(device):
    Hq, Hkv = 32, 8
    lens = np.array([1 << 20, 17, 4096 + 5], np.int64)
    say(f"decode rows of {lens.tolist()} keys, Hq={Hq} Hkv={Hkv}")
    lay, k, v, gen = pools(61, lens, Hkv, device)
    q = synth.randn_bf16((lens.size, Hq, 128), gen, device)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device))
    kl, mk = i32(lens, device), int(lens.max())
    out, lse = ra.decode(q, kv, kl, mk, SCALE, want_lse=True)
    out2 = torch.empty_like(out)
    lse2 = torch.empty_like(lse)
    ra.decode_noalloc(q, kv, kl, mk, out2, SCALE, lse=lse2)
    torch.cuda.synchronize()
    assert torch.equal(out, out2) and torch.equal(lse, lse2), "no-allocation decode differs"
    kk, vv, bt = compact_rows(k, v, lay.block_table, lens)
    ref, ref_lse = oracle.decode(bits(q), kk, vv, bt, lens, SCALE)
    assert_attn_close(out.cpu().numpy(), ref, "decode, a 1,048,576-key row")
    np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, atol=DECODE_LSE_ATOL, rtol=0)


def test_append_after_a_quarter_million_tokens(device):
    Hq, Hkv = 32, 8
    ctx, T = [1 << 18, 0], [300, 7]
    lens = np.array([c + n for c, n in zip(ctx, T)], np.int64)
    say(f"append chunks {T} after contexts {ctx}, Hq={Hq} Hkv={Hkv}")
    lay, k, v, gen = pools(62, lens, Hkv, device)
    cu = np.concatenate([[0], np.cumsum(T)]).astype(np.int32)
    q = synth.randn_bf16((int(cu[-1]), Hq, 128), gen, device)
    kv = ra.PagedKV(k, v, i32(lay.block_table, device))
    out, lse = ra.append(q, i32(cu, device), i32(ctx, device), kv, max(T), int(lens.max()),
                         SCALE, want_lse=True)
    torch.cuda.synchronize()
    # sampled queries: the first, middle and last of the long chunk, all of the short one
    picks = [(0, i) for i in (0, 150, 299)] + [(1, i) for i in range(T[1])]
    sel = [int(cu[r]) + i for r, i in picks]
    kv_len = [ctx[r] + i + 1 for r, i in picks]
    table = lay.block_table[np.array([r for r, _ in picks])]
    kk, vv, bt = compact_rows(k, v, table, np.array(kv_len))
    idx = torch.as_tensor(sel, device=device)
    ref, ref_lse = oracle.decode(bits(q[idx]), kk, vv, bt, kv_len, SCALE)
    assert_attn_close(out[idx].cpu().numpy(), ref, "append after 262,144 tokens (sampled)")
    np.testing.assert_allclose(lse[idx].cpu().numpy(), ref_lse, atol=APPEND_LSE_ATOL, rtol=0)
