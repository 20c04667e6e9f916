"""Calls launched on a side stream with outputs and workspaces the binding allocates.

The binding allocates the call's outputs and workspace with torch while the
kernels run on the caller's stream. It records those blocks on that stream, so
torch's caching allocator must not hand them to work on the current stream
before the kernels are done. The test drops every reference right after each
call and makes the default stream allocate and fill blocks of the same sizes
meanwhile; the results must still equal the default-stream results bitwise and
the oracle within the attention tolerance.
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


def churn(dev, sizes, rounds=6):
    """Allocate and overwrite blocks of the given byte sizes on the current stream."""
    for r in range(rounds):
        held = [torch.full((n,), 0xFF - r, dtype=torch.uint8, device=dev) for n in sizes]
        del held


@pytest.mark.parametrize("handle", ["stream", "int"])
def test_side_stream_decode_and_append_with_binding_allocations(device, handle):
    wd, wa = synth.config(2), synth.config(3)
    print(f"[gpu-test] side stream ({handle}): decode {wd.name}, append {wa.name}", flush=True)
    td, ta = synth.make_tensors(wd, device), synth.make_tensors(wa, device)
    kv_d = ra.PagedKV(td.k_pool, td.v_pool, i32(wd.decode_table(), device))
    kv_a = ra.PagedKV(ta.k_pool, ta.v_pool, i32(wa.append_table(), device))
    kl, cu, ctx = i32(wd.kv_lens, device), i32(wa.cu_q(), device), i32(wa.ctx_lens, device)
    mkd, mq = int(wd.kv_lens.max()), int(wa.q_lens.max())
    mka = int((wa.ctx_lens + wa.q_lens).max())
    # reference results on the default stream
    ref_d, _ = ra.decode(td.q_decode, kv_d, kl, mkd, SCALE)
    ref_a, _ = ra.append(ta.q_append, cu, ctx, kv_a, mq, mka, SCALE)
    torch.cuda.synchronize()
    ws_sizes = [ra.decode_workspace_size(wd.kv_lens.size, wd.Hq, wd.Hkv, mkd),
                ra.append_workspace_size(wa.q_lens.size, wa.Hq, wa.Hkv, mq),
                ref_d.numel() * 4, ref_a.numel() * 4]
    side = torch.cuda.Stream(device)
    arg = side if handle == "stream" else side.cuda_stream
    outs = []
    for _ in range(3):
        od, _ = ra.decode(td.q_decode, kv_d, kl, mkd, SCALE, stream=arg)
        oa, _ = ra.append(ta.q_append, cu, ctx, kv_a, mq, mka, SCALE, stream=arg)
        churn(device, ws_sizes)          # default stream, while the side stream runs
        outs.append((od, oa))
        del od, oa
    side.synchronize()
    torch.cuda.synchronize()
    for od, oa in outs:
        assert torch.equal(od, ref_d), "decode on the side stream differs"
        assert torch.equal(oa, ref_a), "append on the side stream differs"
    rows = sample_rows(wd.kv_lens, 4, seed=5)
    k, v, bt = compact_rows(td.k_pool, td.v_pool, wd.decode_table()[rows], wd.kv_lens[rows])
    want, _ = oracle.decode(bits(td.q_decode[torch.as_tensor(rows, device=device)]), k, v, bt,
                            wd.kv_lens[rows], SCALE)
    assert_attn_close(outs[-1][0][torch.as_tensor(rows, device=device)].cpu().numpy(), want,
                      "side-stream decode, sampled rows")
