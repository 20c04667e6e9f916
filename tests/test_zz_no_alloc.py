"""The no-allocation decode (rollout_attn_decode_noalloc) against rollout_attn_decode.

Both run the same split and combine kernels with the same plan; the only
difference is where the split partials live (the library's per-GPU scratch
instead of a caller workspace), so the outputs must be equal bit for bit. Two
calls in a row, the second on a smaller input, so that the second finds the
first call's partials still in the scratch. Sampled rows are also checked
against the fp64 oracle.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2603_18815_amd as ra
import synth
from tests.gpu_util import DECODE_LSE_ATOL, assert_attn_close, bits, compact_rows, sample_rows

pytestmark = pytest.mark.gpu
SCALE = 1.0 / math.sqrt(128)


def i32(x, dev):
    return torch.as_tensor(np.ascontiguousarray(np.asarray(x, np.int32)), device=dev)


def test_noalloc_decode_equals_decode_on_two_calls(device):
    for c in (2, 1):   # the Qwen3-8B decode workload, then the small one
        w = synth.config(c)
        print(f"[gpu-test] decode_noalloc vs decode: {w.name}", flush=True)
        t = synth.make_tensors(w, device)
        kv = ra.PagedKV(t.k_pool, t.v_pool, i32(w.decode_table(), device))
        kl, mk = i32(w.kv_lens, device), int(w.kv_lens.max())
        B, Hq = w.kv_lens.shape[0], w.Hq
        assert ra.decode_workspace_size(B, Hq, w.Hkv, mk) <= ra._lib.RA_NOALLOC_SCRATCH_BYTES
        ref, ref_lse = ra.decode(t.q_decode, kv, kl, mk, SCALE, want_lse=True)
        out = torch.full((B, Hq, 128), float("nan"), dtype=torch.float32, device=device)
        lse = torch.full((B, Hq), float("nan"), dtype=torch.float32, device=device)
        ra.decode_noalloc(t.q_decode, kv, kl, mk, out, SCALE, lse=lse)
        torch.cuda.synchronize()
        assert torch.equal(out, ref) and torch.equal(lse, ref_lse), w.name
        rows = sample_rows(w.kv_lens, 6, seed=c)
        k, v, bt = compact_rows(t.k_pool, t.v_pool, w.decode_table()[rows], w.kv_lens[rows])
        sel = torch.as_tensor(rows, device=device)
        want, want_lse = oracle.decode(bits(t.q_decode[sel]), k, v, bt, w.kv_lens[rows], SCALE)
        assert_attn_close(out[sel].cpu().numpy(), want, f"decode_noalloc {w.name}")
        np.testing.assert_allclose(lse[sel].cpu().numpy(), want_lse, atol=DECODE_LSE_ATOL, rtol=0)
        del t, kv, out, lse, ref, ref_lse
        torch.cuda.empty_cache()
