"""GPU parity of shared-prefix decode (through the C ABI) against the fp64 CPU oracle.

Rows of a group share their first pages (the rollouts of one task share its
prompt). The oracle is the plain decode definition applied row by row through
each row's own block table, so it checks both the group pass over the shared
keys and the per-row pass over the rest, and the merge of the two.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2603_18815_amd as ra
import synth
from tests.gpu_util import assert_attn_close, bits, compact_rows, sample_rows

pytestmark = pytest.mark.gpu
SCALE = 1.0 / math.sqrt(128)


def i32(x, dev):
    return torch.as_tensor(np.ascontiguousarray(np.asarray(x, np.int32)), device=dev)


def say(msg):
    print(f"[gpu-test] {msg}", flush=True)


def small_groups(seed, sizes, prefix_pages, suffix, Hq, Hkv, dev):
    """A shared-prefix layout with explicit group sizes, prefix pages and suffix lengths."""
    rng = np.random.default_rng(seed)
    pre = np.asarray(prefix_pages, np.int64) * 16
    lay = synth.shared_prefix_layout(rng, sizes, pre, suffix)
    gen = synth.value_generator(seed, dev)
    k = synth.randn_bf16((lay.num_pages, Hkv, 16, 128), gen, dev)
    v = synth.randn_bf16((lay.num_pages, Hkv, 128, 16), gen, dev)
    q = synth.randn_bf16((len(suffix), Hq, 128), gen, dev)
    gs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    return lay, k, v, q, gs, pre.astype(np.int32)


def run_shared(q, k, v, bt, lens, gs, prefix, dev, max_prefix=None):
    kv = ra.PagedKV(k, v, i32(bt, dev))
    sizes = np.diff(gs)
    return ra.decode_shared_prefix(q, kv, i32(lens, dev), i32(gs, dev), i32(prefix, dev),
                                   int(sizes.max()),
                                   int(prefix.max()) if max_prefix is None else max_prefix,
                                   int(np.max(lens)), SCALE, want_lse=True)


@pytest.mark.parametrize("Hq,Hkv,sizes", [
    (32, 8, [8, 8, 8]),        # G = 4: a 16-column tile holds 4 rows, two chunks a group
    (16, 2, [3, 1, 8, 5]),     # G = 8: groups of up to 8 split into 2-row chunks
    (16, 1, [2, 3]),           # G = 16: one row per chunk
    (8, 8, [16, 4]),           # G = 1: one tile holds 16 rows
    (32, 1, [3, 2]),           # G = 32: one row per chunk, two tiles (suffixes too)
    (24, 1, [2, 1]),           # G = 24: two tiles, the second partly empty
    # G = 4, nine ragged groups: the prefix items fill several grid planes, the
    # last one partly
    (32, 8, [5, 8, 3, 1, 7, 2, 8, 4, 6]),
])
def test_shared_prefix_decode_vs_oracle(device, Hq, Hkv, sizes):
    say(f"shared-prefix decode Hq={Hq} Hkv={Hkv} groups={sizes}")
    rng = np.random.default_rng(sum(sizes) + Hq)
    n = sum(sizes)
    # prefixes of 0 pages, 3 pages (48 keys: not a multiple of 32), and longer;
    # suffixes from 1 key to a few splits
    prefix_pages = [[0, 3, 40, 17, 9][i % 5] for i in range(len(sizes))]
    suffix = rng.integers(1, 700, size=n)
    suffix[0] = 1
    lay, k, v, q, gs, pre = small_groups(n + Hq, sizes, prefix_pages, suffix, Hq, Hkv, device)
    lens = lay.row_tokens.astype(np.int32).copy()
    out, lse = run_shared(q, k, v, lay.block_table, lens, gs, pre, device)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.decode(bits(q), bits(k), bits(v), lay.block_table, lens, SCALE)
    assert_attn_close(out.cpu().numpy(), ref, f"shared prefix G={Hq // Hkv}")
    np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, atol=1e-4, rtol=0)


def test_shared_prefix_shorter_row_and_empty_rows(device):
    """A row shorter than its group's prefix caps the shared part; empty rows give 0 / -inf."""
    Hq, Hkv = 8, 2
    lay, k, v, q, gs, pre = small_groups(21, [4, 3], [20, 6], [300, 5, 40, 700, 1, 2, 3],
                                         Hq, Hkv, device)
    lens = lay.row_tokens.astype(np.int32).copy()
    lens[1] = 200          # inside the 320-key prefix of group 0
    lens[5] = 0            # an empty row in group 1 (its shared part becomes 0)
    out, lse = run_shared(q, k, v, lay.block_table, lens, gs, pre, device)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.decode(bits(q), bits(k), bits(v), lay.block_table, lens, SCALE)
    assert torch.all(out[5] == 0) and torch.all(torch.isneginf(lse[5]))
    keep = [r for r in range(len(lens)) if r != 5]
    assert_attn_close(out.cpu().numpy()[keep], ref[keep], "shared prefix, short and empty rows")
    np.testing.assert_allclose(lse.cpu().numpy()[keep], ref_lse[keep], atol=1e-4, rtol=0)


def test_shared_prefix_zero_prefix_is_plain_decode_bitwise(device):
    """With nothing shared the per-row pass is exactly the plain decode's split pass."""
    w = synth.config(1)
    t = synth.make_tensors(w, device)
    kv = ra.PagedKV(t.k_pool, t.v_pool, i32(w.decode_table(), device))
    lens = i32(w.kv_lens, device)
    B = w.kv_lens.size
    a, la = ra.decode(t.q_decode, kv, lens, int(w.kv_lens.max()), SCALE, want_lse=True)
    gs = i32([0, 2, B], device)
    b, lb = ra.decode_shared_prefix(t.q_decode, kv, lens, gs, i32([0, 0], device), B - 2,
                                    min(64, int(w.kv_lens.max())), int(w.kv_lens.max()), SCALE,
                                    want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(la, lb)


def test_shared_prefix_poison_and_determinism(device):
    """NaN in decoy pages and past each row's end is bitwise invisible; repeated calls agree."""
    Hq, Hkv = 32, 8
    sizes = [8, 5]
    suffix = np.array([33, 1, 2, 15, 16, 17, 100, 900, 31, 32, 33, 64, 500])
    lay, k, v, q, gs, pre = small_groups(33, sizes, [7, 12], suffix, Hq, Hkv, device)
    lens = lay.row_tokens.astype(np.int32)
    clean, clean_lse = run_shared(q, k, v, lay.block_table, lens, gs, pre, device)
    again, again_lse = run_shared(q, k, v, lay.block_table, lens, gs, pre, device)
    synth.poison_unowned(k, v, lay)
    dirty, dirty_lse = run_shared(q, k, v, lay.block_table, lens, gs, pre, device)
    torch.cuda.synchronize()
    assert torch.equal(clean, again) and torch.equal(clean_lse, again_lse)
    assert torch.equal(clean, dirty) and torch.equal(clean_lse, dirty_lse)


def test_shared_prefix_workload_sampled(device):
    """The 8 tasks x 8 rollouts workload at full size, sampled rows vs the oracle, and
    against the plain decode of the same rows."""
    w = synth.config(6)
    say(f"shared prefix {w.name}")
    t = synth.make_tensors(w, device)
    bt = w.decode_table()
    out, lse = run_shared(t.q_decode, t.k_pool, t.v_pool, bt, w.kv_lens, w.group_start,
                          w.prefix_len, device)
    kv = ra.PagedKV(t.k_pool, t.v_pool, i32(bt, device))
    plain, plain_lse = ra.decode(t.q_decode, kv, i32(w.kv_lens, device), int(w.kv_lens.max()),
                                 SCALE, want_lse=True)
    torch.cuda.synchronize()
    assert_attn_close(out.cpu().numpy(), plain.cpu().numpy().astype(np.float64),
                      "shared prefix vs plain decode, all rows")
    rows = sample_rows(w.kv_lens, 6, seed=6)
    k, v, btc = compact_rows(t.k_pool, t.v_pool, bt[rows], w.kv_lens[rows])
    ref, ref_lse = oracle.decode(bits(t.q_decode[torch.as_tensor(rows, device=device)]), k, v,
                                 btc, w.kv_lens[rows], SCALE)
    sel = torch.as_tensor(rows, device=device)
    assert_attn_close(out[sel].cpu().numpy(), ref, f"{w.name} sampled rows")
    np.testing.assert_allclose(lse[sel].cpu().numpy(), ref_lse, atol=1e-4, rtol=0)
