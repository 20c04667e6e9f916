"""Host logic of bench.py (CPU only): the one-GPU guard, the algorithmic work
counts that every reported rate divides by, and the rule that a traffic figure
is reported only while the kernel sources match the profile it came from."""
import hashlib
import os
import subprocess
import sys
from types import SimpleNamespace

import numpy as np

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_decode_bytes_counts_every_key_once():
    """Per row: each attended key's K and V of every KV head (bf16), q in bf16,
    out in fp32, one table entry per page and the length."""
    for c in (1, 2):
        w = synth.config(c)
        total = 0
        for L in w.kv_lens.tolist():
            total += sum(w.Hkv * w.head_dim * 2 * 2 for _ in range(L))
            total += w.Hq * w.head_dim * (2 + 4)
            total += 4 * len(range(0, L, w.page_size)) + 4
        assert bench.decode_bytes(w) == total


def test_append_flops_count_unmasked_pairs():
    """4 * D * Hq flops per (query, key) pair that the causal mask keeps, counted
    by enumerating the pairs of small rows."""
    rng = np.random.default_rng(3)
    T = rng.integers(0, 40, size=9)
    C = rng.integers(0, 70, size=9)
    T[0], C[1] = 0, 0                      # an empty chunk, a chunk with no cached context
    w = SimpleNamespace(q_lens=T, ctx_lens=C, Hq=32, head_dim=128)
    pairs = sum(1 for t, c in zip(T, C) for i in range(t) for j in range(c + t) if j <= c + i)
    assert bench.append_flops(w) == 4 * 128 * 32 * pairs
    w3 = synth.config(3)
    assert bench.append_flops(w3) == int(4 * 128 * w3.Hq * sum(
        int(t) * int(c) + int(t) * (int(t) + 1) // 2 for t, c in zip(w3.q_lens, w3.ctx_lens)))


def test_write_bytes():
    # read and write of K and V, bf16, Hkv heads of 128 dims per new token
    assert bench.write_bytes(10, 8) == 10 * 8 * 128 * 2 * 2 * 2


def test_traffic_reported_only_for_matching_sources(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("kernel v1\n")
    digest = hashlib.sha256(src.read_bytes()).hexdigest()[:16]
    prof = tmp_path / "t.txt"
    prof.write_text(f"# header = not a field\nhbm_bytes_per_launch = 1234.0\n"
                    f"source_sha256_16 = {digest}   # k.hip\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "KERNEL_SOURCES", {"decode": ("k.hip",)})
    monkeypatch.setattr(bench, "TRAFFIC_FILES", {"decode": "t.txt"})
    assert bench.measured_traffic("decode") == 1234
    src.write_text("kernel v2\n")                      # the kernel changed since profiling
    assert bench.measured_traffic("decode") is None
    prof.unlink()
    assert bench.measured_traffic("decode") is None


def test_committed_traffic_files_name_their_sources():
    """Every committed traffic summary records the hash of the sources bench.py
    checks for it, in the form measured_traffic parses."""
    for part, rel in bench.TRAFFIC_FILES.items():
        fields = {}
        for line in open(os.path.join(ROOT, rel)):
            if "=" in line and not line.startswith("#"):
                k, v = line.split("#")[0].split("=", 1)
                fields[k.strip()] = v.strip()
        assert float(fields["hbm_bytes_per_launch"]) > 0, part
        assert len(fields["source_sha256_16"]) == 16, part
