"""Seeded input generator: determinism and layout well-formedness (CPU only)."""
import numpy as np
import torch

import synth


def test_layouts_are_deterministic_and_well_formed():
    for c in (1, 2, 3, 4, 5):
        w1, w2 = synth.config(c), synth.config(c)
        np.testing.assert_array_equal(w1.layout.block_table, w2.layout.block_table)
        lay = w1.layout
        P = w1.page_size
        pages = (lay.row_tokens.astype(np.int64) + P - 1) // P
        owned = np.concatenate([lay.block_table[b, :pages[b]] for b in range(len(pages))])
        # every owned page appears once; decoys are never owned; ids are in range
        assert len(np.unique(owned)) == owned.size
        assert np.intersect1d(owned, lay.decoys).size == 0
        assert owned.size + lay.decoys.size == lay.num_pages
        assert lay.block_table.min() >= 0 and lay.block_table.max() < lay.num_pages
        assert lay.decoys.size >= 16


def test_workload_ranges():
    w = synth.config(2)
    assert w.kv_lens.min() >= 4096 and w.kv_lens.max() <= 32768 and w.G == 4
    w = synth.config(3)
    assert w.ctx_lens.min() >= 2048 and w.ctx_lens.max() <= 24576
    assert w.q_lens.min() >= 64 and w.q_lens.max() <= 2048
    w = synth.config(4)
    assert w.kv_lens.min() >= 512 and w.kv_lens.max() <= 65536 and w.G == 8
    w = synth.config(5)
    assert w.decode_rows.size + w.append_rows.size == 512 and w.append_rows.size == 77
    assert np.intersect1d(w.decode_rows, w.append_rows).size == 0


def test_values_are_deterministic_bf16_normal():
    w = synth.config(1)
    t1 = synth.make_tensors(w, "cpu")
    t2 = synth.make_tensors(w, "cpu")
    assert torch.equal(t1.k_pool, t2.k_pool) and torch.equal(t1.q_decode, t2.q_decode)
    assert t1.k_pool.dtype == torch.bfloat16
    assert t1.k_pool.shape == (w.layout.num_pages, 2, 16, 128)
    assert t1.v_pool.shape == (w.layout.num_pages, 2, 128, 16)
    x = t1.k_pool.float()
    assert abs(x.mean().item()) < 0.05 and abs(x.std().item() - 1.0) < 0.05


def test_write_plan_positions():
    w = synth.config(5)
    bt, cu, start = synth.write_plan(w)
    nd = w.decode_rows.size
    assert np.all(np.diff(cu[:nd + 1]) == 1)
    np.testing.assert_array_equal(start[:nd], w.kv_lens - 1)
    np.testing.assert_array_equal(start[nd:], w.ctx_lens)
    np.testing.assert_array_equal(np.diff(cu[nd:]), w.q_lens)


def test_poison_marks_decoys_and_tails():
    w = synth.config(1)
    t = synth.make_tensors(w, "cpu")
    synth.poison_unowned(t.k_pool, t.v_pool, w.layout)
    dec = torch.as_tensor(w.layout.decoys.astype(np.int64))
    assert torch.isnan(t.k_pool[dec].float()).all() and torch.isnan(t.v_pool[dec].float()).all()
    for b, L in enumerate(w.layout.row_tokens):
        pg = w.layout.block_table[b, (L - 1) // 16]
        assert not torch.isnan(t.k_pool[pg, :, (L - 1) % 16].float()).any()
        if L % 16:
            assert torch.isnan(t.k_pool[pg, :, L % 16:].float()).all()


def test_shared_prefix_layout():
    w = synth.config(6)
    lay, P = w.layout, w.page_size
    assert w.group_start.tolist() == list(range(0, 65, 8)) and w.G == 4
    assert np.all(w.prefix_len % P == 0) and w.prefix_len.min() >= 2048
    assert np.all(w.kv_lens - np.repeat(w.prefix_len, 8) >= 2048)
    owned = []
    for i in range(w.prefix_len.size):
        rows = range(w.group_start[i], w.group_start[i + 1])
        n = w.prefix_len[i] // P
        shared = lay.block_table[rows[0], :n]
        for r in rows:       # every row of a group maps its prefix to the same pages
            np.testing.assert_array_equal(lay.block_table[r, :n], shared)
            owned.append(lay.block_table[r, n:(w.kv_lens[r] + P - 1) // P])
        owned.append(shared)
    owned = np.concatenate(owned)
    # shared pages once per group, suffix pages once per row, decoys never owned
    assert len(np.unique(owned)) == owned.size
    assert np.intersect1d(owned, lay.decoys).size == 0
    assert owned.size + lay.decoys.size == lay.num_pages
