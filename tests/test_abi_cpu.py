"""C ABI checks that need no GPU: the library loads, exports every declared
symbol, and rejects bad arguments before touching HIP (CPU only)."""
import ctypes
import os
import re

import pytest

from paper_2603_18815_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rollout_attn.h")

FAKE = 0x1000  # never dereferenced: every call below fails validation first


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)))


def _kv(**kw):
    d = dict(k_pool=FAKE, v_pool=FAKE, block_table=FAKE, num_pages=10, bt_stride=4,
             num_kv_heads=2, page_size=16, head_dim=128, kv_dtype=_lib.RA_KV_BF16, k_scale=1.0,
             v_scale=1.0)
    d.update(kw)
    return _lib.RaPagedKV(**d)


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def test_exports_every_declared_symbol(lib):
    names = _declared_functions()
    assert set(names) == set(_lib.EXPORTS), names
    for n in names:
        assert hasattr(lib, n), n


def test_abi_version_and_status_strings(lib):
    declared = int(re.search(r"#define RA_ABI_VERSION (\d+)", open(HEADER).read()).group(1))
    assert lib.ra_abi_version() == declared == 6
    assert lib.ra_status_string(0) == b"RA_OK"
    assert lib.ra_status_string(4) == b"RA_ERR_WORKSPACE"
    assert lib.ra_status_string(99) == b"RA_UNKNOWN_STATUS"


def test_workspace_size(lib):
    f = lib.rollout_attn_decode_workspace_size
    assert f(0, 32, 8, 1000) == 0
    a = f(64, 32, 8, 32768)
    assert a > 0 and a % 4 == 0
    assert f(64, 32, 8, 65536) >= a          # longer rows need at least as many splits
    assert f(128, 32, 8, 32768) >= a


def _decode(lib, kv, **kw):
    d = dict(q=FAKE, kv_lens=FAKE, B=2, Hq=4, max_kv_len=64, scale=0.1, out=FAKE, lse=None,
             ws=FAKE, ws_bytes=1 << 30, stream=None)
    d.update(kw)
    return lib.rollout_attn_decode(d["q"], ctypes.byref(kv), d["kv_lens"], d["B"], d["Hq"],
                                   d["max_kv_len"], d["scale"], d["out"], d["lse"], d["ws"],
                                   d["ws_bytes"], d["stream"])


def test_decode_validation(lib):
    assert _decode(lib, _kv(), q=None) == _lib.RA_ERR_NULL
    assert _decode(lib, _kv(), out=None) == _lib.RA_ERR_NULL
    assert _decode(lib, _kv(k_pool=None)) == _lib.RA_ERR_NULL
    assert _decode(lib, _kv(), B=-1) == _lib.RA_ERR_SHAPE
    assert _decode(lib, _kv(), Hq=3) == _lib.RA_ERR_SHAPE                 # Hq % Hkv
    assert _decode(lib, _kv(), max_kv_len=65) == _lib.RA_ERR_SHAPE        # > bt_stride * 16
    assert _decode(lib, _kv(page_size=32)) == _lib.RA_ERR_UNSUPPORTED
    assert _decode(lib, _kv(head_dim=64)) == _lib.RA_ERR_UNSUPPORTED
    assert _decode(lib, _kv(), Hq=66) == _lib.RA_ERR_UNSUPPORTED          # group of 33
    assert _decode(lib, _kv(), Hq=64, B=0) == _lib.RA_OK                  # group of 32
    assert _decode(lib, _kv(), ws_bytes=16) == _lib.RA_ERR_WORKSPACE
    assert _decode(lib, _kv(), ws=None) == _lib.RA_ERR_WORKSPACE
    assert _decode(lib, _kv(), B=0) == _lib.RA_OK                         # no work, no launch


def test_shared_prefix_decode_validation(lib):
    def call(kv=None, **kw):
        d = dict(q=FAKE, kv_lens=FAKE, gs=FAKE, pre=FAKE, B=16, Hq=4, ng=2, mgr=8, mpl=32,
                 max_kv_len=64, out=FAKE, ws=FAKE, ws_bytes=1 << 30)
        d.update(kw)
        return lib.rollout_attn_decode_shared_prefix(
            d["q"], ctypes.byref(kv if kv is not None else _kv()), d["kv_lens"], d["gs"],
            d["pre"], d["B"], d["Hq"], d["ng"], d["mgr"], d["mpl"], d["max_kv_len"], 0.1,
            d["out"], None, d["ws"], d["ws_bytes"], None)
    assert call(gs=None) == _lib.RA_ERR_NULL
    assert call(pre=None) == _lib.RA_ERR_NULL
    assert call(ng=-1) == _lib.RA_ERR_SHAPE
    assert call(ng=0) == _lib.RA_ERR_SHAPE           # rows must belong to groups
    assert call(mgr=0) == _lib.RA_ERR_SHAPE
    assert call(mgr=17) == _lib.RA_ERR_SHAPE         # more rows per group than rows
    assert call(mpl=65) == _lib.RA_ERR_SHAPE         # prefix bound above max_kv_len
    assert call(Hq=5) == _lib.RA_ERR_SHAPE
    assert call(Hq=66) == _lib.RA_ERR_UNSUPPORTED    # group of 33 query heads
    assert call(ws_bytes=16) == _lib.RA_ERR_WORKSPACE
    assert call(ws=None) == _lib.RA_ERR_WORKSPACE
    big = dict(B=65535, ng=65535, mgr=2, max_kv_len=64)
    assert call(**big) == _lib.RA_ERR_UNSUPPORTED    # grid of groups x rows too large
    # the row planes alone fit (65,535), the prefix items' planes push the grid past it
    assert call(B=65535, ng=1, mgr=65535, mpl=16, max_kv_len=32) == _lib.RA_ERR_UNSUPPORTED
    assert call(B=0) == _lib.RA_OK
    f = lib.rollout_attn_decode_shared_prefix_workspace_size
    plain = lib.rollout_attn_decode_workspace_size(64, 32, 8, 32768)
    assert f(64, 32, 8, 32768, 0) == plain           # no prefix slots
    assert f(64, 32, 8, 32768, 8192) > plain         # plus the prefix slots
    assert f(0, 32, 8, 32768, 8192) == 0


def test_token_logprob_validation(lib):
    def call(**kw):
        d = dict(h=FAKE, W=FAKE, t=FAKE, N=8, V=100, D=128, out=FAKE, ws=FAKE, ws_bytes=1 << 30)
        d.update(kw)
        return lib.token_logprob(d["h"], d["W"], d["t"], d["N"], d["V"], d["D"], 1.0, d["out"],
                                 None, d["ws"], d["ws_bytes"], None)
    assert call(h=None) == _lib.RA_ERR_NULL
    assert call(out=None) == _lib.RA_ERR_NULL
    assert call(N=-1) == _lib.RA_ERR_SHAPE
    assert call(V=0) == _lib.RA_ERR_SHAPE
    assert call(D=0) == _lib.RA_ERR_SHAPE
    assert call(D=96) == _lib.RA_ERR_UNSUPPORTED       # not a multiple of 64
    assert call(ws_bytes=4) == _lib.RA_ERR_WORKSPACE
    assert call(N=0) == _lib.RA_OK
    f = lib.token_logprob_workspace_size
    assert f(0, 100, 128) == 0 and f(8, 0, 128) == 0
    assert f(8, 100, 0) == 0 and f(8, 100, 96) == 0      # D not a positive multiple of 64
    assert f(64, 151936, 4096) == (64 * 1187 * 2 + 64) * 4     # 1187 chunks of 128 rows
    assert f(511, 151936, 4096) == (511 * 1187 * 2 + 511) * 4
    # from N = 512: 396 chunks of 384 rows, then (at a 256-byte boundary) the
    # staged copy of h, N rounded up to whole 256-token blocks
    for N, padded in ((512, 512), (513, 768)):
        part = (N * 396 * 2 + N) * 4
        assert f(N, 151936, 4096) == (part + 255) // 256 * 256 + padded * 4096 * 2


def test_token_logprob_packed_validation(lib):
    size = lib.token_logprob_packed_weight_size
    assert size(151936, 4096) == 396 * 384 * 4096 * 2    # V rounded up to 384 rows
    assert size(1, 64) == 384 * 64 * 2
    assert size(0, 64) == 0 and size(10, 0) == 0 and size(10, 96) == 0
    # the largest V: the rounding to whole 384-row chunks must not overflow
    big = 2**31 - 1
    assert size(big, 64) == (big + 383) // 384 * 384 * 64 * 2
    assert lib.token_logprob_workspace_size(1, big, 64) == ((big + 127) // 128 * 2 + 1) * 4
    assert lib.token_logprob_workspace_size(512, big, 64) == \
        ((512 * ((big + 383) // 384) * 2 + 512) * 4 + 255) // 256 * 256 + 512 * 64 * 2

    def pack(**kw):
        d = dict(W=FAKE, V=100, D=128, Wp=FAKE, nbytes=1 << 30)
        d.update(kw)
        return lib.token_logprob_pack_weight(d["W"], d["V"], d["D"], d["Wp"], d["nbytes"], None)
    assert pack(W=None) == _lib.RA_ERR_NULL
    assert pack(Wp=None) == _lib.RA_ERR_NULL
    assert pack(V=0) == _lib.RA_ERR_SHAPE
    assert pack(D=-64) == _lib.RA_ERR_SHAPE
    assert pack(D=96) == _lib.RA_ERR_UNSUPPORTED
    assert pack(nbytes=384 * 128 * 2 - 1) == _lib.RA_ERR_WORKSPACE

    def call(**kw):
        d = dict(h=FAKE, W=FAKE, t=FAKE, N=8, V=100, D=128, out=FAKE, ws=FAKE, ws_bytes=1 << 30)
        d.update(kw)
        return lib.token_logprob_packed(d["h"], d["W"], d["t"], d["N"], d["V"], d["D"], 1.0,
                                        d["out"], None, d["ws"], d["ws_bytes"], None)
    assert call(W=None) == _lib.RA_ERR_NULL
    assert call(t=None) == _lib.RA_ERR_NULL
    assert call(N=-1) == _lib.RA_ERR_SHAPE
    assert call(V=0) == _lib.RA_ERR_SHAPE
    assert call(D=96) == _lib.RA_ERR_UNSUPPORTED
    assert call(ws_bytes=4) == _lib.RA_ERR_WORKSPACE
    assert call(N=0) == _lib.RA_OK


def test_append_validation(lib):
    def call(kv, **kw):
        d = dict(q=FAKE, cu=FAKE, ctx=FAKE, B=2, Hq=4, total_q=10, max_q=5, max_kv=64,
                 out=FAKE, ws=FAKE, ws_bytes=1 << 30)
        d.update(kw)
        return lib.rollout_attn_append(d["q"], d["cu"], d["ctx"], ctypes.byref(kv), d["B"],
                                       d["Hq"], d["total_q"], d["max_q"], d["max_kv"], 0.1,
                                       d["out"], None, d["ws"], d["ws_bytes"], None)
    assert call(_kv(), cu=None) == _lib.RA_ERR_NULL
    assert call(_kv(), total_q=-1) == _lib.RA_ERR_SHAPE
    assert call(_kv(), max_kv=100) == _lib.RA_ERR_SHAPE
    assert call(_kv(), max_q=70, max_kv=64) == _lib.RA_ERR_SHAPE
    assert call(_kv(), Hq=5) == _lib.RA_ERR_SHAPE
    assert call(_kv(head_dim=256)) == _lib.RA_ERR_UNSUPPORTED
    assert call(_kv(), ws_bytes=16) == _lib.RA_ERR_WORKSPACE
    assert call(_kv(), ws=None) == _lib.RA_ERR_WORKSPACE
    assert call(_kv(num_kv_heads=512), Hq=512) == _lib.RA_ERR_UNSUPPORTED   # > 256 KV heads
    assert call(_kv(), total_q=0, ws=None) == _lib.RA_OK                   # no work, no launch
    assert call(_kv(), B=0, ws=None) == _lib.RA_OK


def test_append_workspace_size(lib):
    f = lib.rollout_attn_append_workspace_size
    assert f(0, 32, 8, 100) == 0
    assert f(4, 30, 8, 100) == 0                                  # Hq % Hkv
    a = f(32, 32, 8, 2048)
    assert a >= 32 * (2048 // 64) * 8 * 8                         # one 8-byte entry per tile
    assert f(32, 32, 8, 4096) > a
    assert f(32, 32, 8, 2048) == lib.rollout_attn_mixed_workspace_size(0, 32, 32, 8, 8, 0, 2048)
    # the largest chunk length: query blocks are counted without overflow
    big = f(1, 32, 8, 2**31 - 1)
    assert big >= ((2**31 - 1 + 63) // 64) * 8 * 8 and big > f(1, 32, 8, 2**30)


def test_page_write_and_gather_validation(lib):
    kv = _kv()
    w = lambda **kw: lib.kv_page_write(kw.get("k", FAKE), FAKE, FAKE, FAKE, ctypes.byref(
        kw.get("kv", kv)), kw.get("B", 2), kw.get("total", 8), kw.get("max_new", 4),
        kw.get("max_pos", 64), None)
    assert w(k=None) == _lib.RA_ERR_NULL
    assert w(max_pos=65) == _lib.RA_ERR_SHAPE
    assert w(max_new=70) == _lib.RA_ERR_SHAPE
    assert w(kv=_kv(num_kv_heads=0)) == _lib.RA_ERR_SHAPE
    assert w(total=0) == _lib.RA_OK
    g = lambda **kw: lib.kv_page_gather(ctypes.byref(kw.get("kv", kv)), FAKE, FAKE,
                                        kw.get("B", 2), 8, kw.get("max_len", 64),
                                        kw.get("k", FAKE), FAKE, None)
    assert g(k=None) == _lib.RA_ERR_NULL
    assert g(max_len=100) == _lib.RA_ERR_SHAPE
    assert g(kv=_kv(page_size=8)) == _lib.RA_ERR_UNSUPPORTED
    assert g(B=0) == _lib.RA_OK


def _mixed(lib, kvd, kva, **kw):
    d = dict(qd=FAKE, kv_lens=FAKE, Bd=2, mkd=64, outd=FAKE, lsed=None,
             qa=FAKE, cu_q=FAKE, ctx=FAKE, Ba=2, total_q=10, mq=8, mka=64, outa=FAKE, lsea=None,
             Hq=4, scale=0.1, ws=FAKE, ws_bytes=1 << 30, stream=None)
    d.update(kw)
    return lib.rollout_attn_mixed(
        d["qd"], None if kvd is None else ctypes.byref(kvd), d["kv_lens"], d["Bd"], d["mkd"],
        d["outd"], d["lsed"], d["qa"], d["cu_q"], d["ctx"],
        None if kva is None else ctypes.byref(kva), d["Ba"], d["total_q"], d["mq"], d["mka"],
        d["outa"], d["lsea"], d["Hq"], d["scale"], d["ws"], d["ws_bytes"], d["stream"])


def test_mixed_workspace_size(lib):
    f = lib.rollout_attn_mixed_workspace_size
    assert f(-1, 2, 32, 8, 8, 1000, 100) == 0
    assert f(4, 4, 30, 8, 8, 1000, 100) == 0             # Hq % Hkv
    a = f(64, 8, 32, 8, 8, 32768, 2048)
    # at least the decode partials, plus the work lists
    assert a > lib.rollout_attn_decode_workspace_size(64, 32, 8, 32768)
    assert f(64, 8, 32, 8, 8, 32768, 4096) > a            # more query blocks, longer tile list
    assert f(0, 8, 32, 8, 8, 0, 2048) > 0                 # append only
    assert f(64, 0, 32, 8, 8, 32768, 0) > 0               # decode only


def test_mixed_validation(lib):
    kv = _kv()
    assert _mixed(lib, kv, kv, qd=None) == _lib.RA_ERR_NULL
    assert _mixed(lib, kv, kv, cu_q=None) == _lib.RA_ERR_NULL
    assert _mixed(lib, None, kv) == _lib.RA_ERR_NULL
    assert _mixed(lib, kv, None) == _lib.RA_ERR_NULL
    assert _mixed(lib, kv, kv, Bd=-1) == _lib.RA_ERR_SHAPE
    assert _mixed(lib, kv, kv, total_q=-1) == _lib.RA_ERR_SHAPE
    assert _mixed(lib, kv, kv, Hq=3) == _lib.RA_ERR_SHAPE                # Hq % Hkv
    assert _mixed(lib, kv, kv, mkd=65) == _lib.RA_ERR_SHAPE              # > bt_stride * 16
    assert _mixed(lib, kv, kv, mq=65, mka=64) == _lib.RA_ERR_SHAPE       # chunk > max_kv_len
    assert _mixed(lib, kv, kv, Hq=66) == _lib.RA_ERR_UNSUPPORTED         # decode group of 33
    assert _mixed(lib, kv, _kv(page_size=32)) == _lib.RA_ERR_UNSUPPORTED
    assert _mixed(lib, kv, _kv(num_kv_heads=512, num_pages=10), Hq=512,
                  Bd=0) == _lib.RA_ERR_UNSUPPORTED                       # > 256 KV heads
    assert _mixed(lib, kv, kv, ws_bytes=16) == _lib.RA_ERR_WORKSPACE
    assert _mixed(lib, kv, kv, ws=None) == _lib.RA_ERR_WORKSPACE
    # an empty side is not checked at all; both empty: no work, no launch
    assert _mixed(lib, None, None, Bd=0, Ba=0, qd=None, qa=None) == _lib.RA_OK
    assert _mixed(lib, kv, None, Bd=0, total_q=0, ws=None) == _lib.RA_OK


def test_fp8_pool_validation(lib):
    """fp8 pools: an unknown element type, bad scales, and the entry points that do not
    take fp8 pools are rejected before any launch."""
    fp8 = dict(kv_dtype=_lib.RA_KV_FP8_E4M3, k_scale=0.5, v_scale=2.0)
    assert _decode(lib, _kv(kv_dtype=7)) == _lib.RA_ERR_UNSUPPORTED
    for bad in (0.0, -1.0, float("inf"), float("nan"), 1e-39):   # 1e-39: 1 / scale overflows
        assert _decode(lib, _kv(**dict(fp8, k_scale=bad))) == _lib.RA_ERR_SHAPE
        assert _decode(lib, _kv(**dict(fp8, v_scale=bad))) == _lib.RA_ERR_SHAPE
    assert _decode(lib, _kv(**fp8), ws_bytes=16) == _lib.RA_ERR_WORKSPACE   # fp8 decode passes
    assert _decode(lib, _kv(**fp8), B=0) == _lib.RA_OK
    # fp8 append passes the element-type check (and fails on the workspace here)
    assert lib.rollout_attn_append(FAKE, FAKE, FAKE, ctypes.byref(_kv(**fp8)), 2, 4, 10, 5, 64,
                                   0.1, FAKE, None, FAKE, 16, None) == _lib.RA_ERR_WORKSPACE
    kv = _kv()
    # a mixed call takes one element type for both sides
    assert _mixed(lib, _kv(**fp8), kv) == _lib.RA_ERR_UNSUPPORTED
    assert _mixed(lib, kv, _kv(**fp8)) == _lib.RA_ERR_UNSUPPORTED
    assert _mixed(lib, _kv(**fp8), _kv(**fp8), ws_bytes=16) == _lib.RA_ERR_WORKSPACE
    # the bf16 scales are ignored
    assert _decode(lib, _kv(k_scale=0.0, v_scale=float("nan")), B=0) == _lib.RA_OK


def test_nonfinite_scale_rejected(lib):
    """Every entry point that takes a softmax or logit scale rejects a
    non-finite one before any launch (finite scales of any sign pass)."""
    for bad in (float("inf"), float("-inf"), float("nan")):
        assert _decode(lib, _kv(), scale=bad) == _lib.RA_ERR_SHAPE
        assert lib.rollout_attn_append(FAKE, FAKE, FAKE, ctypes.byref(_kv()), 2, 4, 10, 5, 64,
                                       bad, FAKE, None, FAKE, 1 << 30, None) == _lib.RA_ERR_SHAPE
        assert lib.rollout_attn_append_write(FAKE, FAKE, FAKE, FAKE, FAKE, ctypes.byref(_kv()),
                                             2, 4, 10, 5, 64, bad, FAKE, None, FAKE, 1 << 30,
                                             None) == _lib.RA_ERR_SHAPE
        assert lib.rollout_attn_decode_shared_prefix(
            FAKE, ctypes.byref(_kv()), FAKE, FAKE, FAKE, 16, 4, 2, 8, 32, 64, bad, FAKE, None,
            FAKE, 1 << 30, None) == _lib.RA_ERR_SHAPE
        assert _mixed(lib, _kv(), _kv(), scale=bad) == _lib.RA_ERR_SHAPE
        assert lib.token_logprob(FAKE, FAKE, FAKE, 8, 100, 128, bad, FAKE, None, FAKE, 1 << 30,
                                 None) == _lib.RA_ERR_SHAPE
        assert lib.token_logprob_packed(FAKE, FAKE, FAKE, 8, 100, 128, bad, FAKE, None, FAKE,
                                        1 << 30, None) == _lib.RA_ERR_SHAPE
    for ok in (0.0, -0.5):
        assert _decode(lib, _kv(), scale=ok, B=0) == _lib.RA_OK


def test_append_write_validation(lib):
    def call(kv, **kw):
        d = dict(q=FAKE, k=FAKE, v=FAKE, cu=FAKE, ctx=FAKE, B=2, Hq=4, total_q=10, max_q=5,
                 max_kv=64, out=FAKE, ws=FAKE, ws_bytes=1 << 30)
        d.update(kw)
        return lib.rollout_attn_append_write(d["q"], d["k"], d["v"], d["cu"], d["ctx"],
                                             ctypes.byref(kv), d["B"], d["Hq"], d["total_q"],
                                             d["max_q"], d["max_kv"], 0.1, d["out"], None,
                                             d["ws"], d["ws_bytes"], None)
    assert call(_kv(), k=None) == _lib.RA_ERR_NULL
    assert call(_kv(), v=None) == _lib.RA_ERR_NULL
    assert call(_kv(), max_kv=100) == _lib.RA_ERR_SHAPE
    assert call(_kv(), Hq=5) == _lib.RA_ERR_SHAPE
    # fp8 pools are accepted (their scales are validated like everywhere else)
    fp8 = dict(kv_dtype=_lib.RA_KV_FP8_E4M3, v_scale=1.0)
    assert call(_kv(k_scale=0.0, **fp8)) == _lib.RA_ERR_SHAPE
    assert call(_kv(k_scale=1.0, **fp8), ws_bytes=16) == _lib.RA_ERR_WORKSPACE
    assert call(_kv(k_scale=1.0, **fp8), total_q=0, ws=None) == _lib.RA_OK
    assert call(_kv(), ws_bytes=16) == _lib.RA_ERR_WORKSPACE
    assert call(_kv(), total_q=0, ws=None) == _lib.RA_OK


def test_plain_c_caller(tmp_path):
    """The header is valid C99 on its own and a C program links the library:
    tests/c_abi_check.c calls every entry point (host-side rejections only)."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    rocm_inc = "/opt/rocm/include"
    if gcc is None or not os.path.isdir(rocm_inc):
        pytest.skip("gcc or the ROCm headers are not available")
    libdir = os.path.dirname(_lib.LIB_PATH)
    exe = tmp_path / "c_abi_check"
    cmd = [gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", rocm_inc,
           os.path.join(ROOT, "tests", "c_abi_check.c"), "-L", libdir, "-lrollout_attn",
           f"-Wl,-rpath,{libdir}", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok (0 failed)"), r.stdout + r.stderr


def test_rope_validation(lib):
    """The rotary variants check their table before anything else of theirs:
    NULL table, no rows, or fewer rows than positions the call uses."""
    def write(**kw):
        d = dict(cs=FAKE, rows=64, B=2, total=4, max_new=2, max_pos=64)
        d.update(kw)
        return lib.kv_page_write_rope(FAKE, FAKE, FAKE, FAKE, ctypes.byref(_kv()), d["B"],
                                      d["total"], d["max_new"], d["max_pos"], d["cs"],
                                      d["rows"], None)
    assert write(cs=None) == _lib.RA_ERR_NULL
    assert write(rows=0) == _lib.RA_ERR_SHAPE
    assert write(rows=63) == _lib.RA_ERR_SHAPE          # positions up to 63 need 64 rows
    assert write(max_pos=65, rows=65) == _lib.RA_ERR_SHAPE   # beyond bt_stride * 16 = 64
    assert write(B=0) == _lib.RA_OK

    def fused(**kw):
        d = dict(cs=FAKE, rows=64, max_kv=64, ws_bytes=1 << 30, total_q=10)
        d.update(kw)
        return lib.rollout_attn_append_write_rope(
            FAKE, FAKE, FAKE, FAKE, FAKE, ctypes.byref(_kv()), 2, 4, d["total_q"], 5,
            d["max_kv"], 0.1, d["cs"], d["rows"], FAKE, None, FAKE, d["ws_bytes"], None)
    assert fused(cs=None) == _lib.RA_ERR_NULL
    assert fused(rows=-1) == _lib.RA_ERR_SHAPE
    assert fused(rows=60) == _lib.RA_ERR_SHAPE          # max_kv_len 64 needs 64 rows
    assert fused(ws_bytes=16) == _lib.RA_ERR_WORKSPACE
    assert fused(total_q=0) == _lib.RA_OK


def _decode_ws_sizes(env_value):
    """Decode workspace sizes computed in a fresh process (the split override is
    read once per process) with RA_SPLIT_TOKENS set to env_value (None: unset)."""
    import subprocess
    import sys
    code = ("import sys; sys.path.insert(0, %r); from paper_2603_18815_amd import _lib; "
            "f = _lib.load().rollout_attn_decode_workspace_size; "
            "print(f(64, 32, 8, 32768), f(2, 8, 2, 1000), f(1, 1, 1, 65536))" % ROOT)
    env = dict(os.environ)
    env.pop("RA_SPLIT_TOKENS", None)
    if env_value is not None:
        env["RA_SPLIT_TOKENS"] = env_value
    out = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                         timeout=120, check=True).stdout.split()
    return tuple(int(v) for v in out)


def test_split_override_is_bounded():
    """RA_SPLIT_TOKENS forces the decode split length only for values in
    [128, 65536] (rounded up to a multiple of 128); anything else - too large for
    an int32, negative, below 128, not a number - leaves the planned split, so
    the workspace size (and the split arithmetic) stays that of no override."""
    def expect(B, Hq, Hkv, L, split):
        return B * Hq * max(1, -(-L // split)) * (128 + 2) * 4

    planned = _decode_ws_sizes(None)
    for bad in ("4294967296", "9223372036854775807", "-512", "127", "65537", "12x", "", "abc"):
        assert _decode_ws_sizes(bad) == planned, bad
    # in range: the split is the value rounded up to a multiple of 128
    assert _decode_ws_sizes("128") == (expect(64, 32, 8, 32768, 128), expect(2, 8, 2, 1000, 128),
                                       expect(1, 1, 1, 65536, 128))
    assert _decode_ws_sizes("200") == (expect(64, 32, 8, 32768, 256), expect(2, 8, 2, 1000, 256),
                                       expect(1, 1, 1, 65536, 256))
    assert _decode_ws_sizes("65536") == (expect(64, 32, 8, 32768, 65536),
                                         expect(2, 8, 2, 1000, 65536),
                                         expect(1, 1, 1, 65536, 65536))


def test_decode_noalloc_validation(lib):
    """The no-allocation decode checks arguments like decode and refuses, before
    any HIP call, plans whose split partials exceed its scratch."""
    f = lib.rollout_attn_decode_noalloc
    kv = _kv()
    assert f(None, ctypes.byref(kv), FAKE, 2, 4, 64, 0.1, FAKE, None, None) == _lib.RA_ERR_NULL
    assert f(FAKE, ctypes.byref(kv), FAKE, 2, 4, 64, 0.1, None, None, None) == _lib.RA_ERR_NULL
    assert f(FAKE, ctypes.byref(kv), FAKE, 2, 5, 64, 0.1, FAKE, None, None) == _lib.RA_ERR_SHAPE
    assert f(FAKE, ctypes.byref(kv), FAKE, 0, 4, 64, 0.1, FAKE, None, None) == _lib.RA_OK
    big = _kv(num_kv_heads=8, bt_stride=4096)
    need = lib.rollout_attn_decode_workspace_size(256, 64, 8, 65536)
    assert need > _lib.RA_NOALLOC_SCRATCH_BYTES
    assert f(FAKE, ctypes.byref(big), FAKE, 256, 64, 65536, 0.1, FAKE, None,
             None) == _lib.RA_ERR_WORKSPACE
    # the Qwen3-8B decode workload (64 rows, 32 heads, up to 32768 keys) fits
    assert lib.rollout_attn_decode_workspace_size(64, 32, 8, 32768) <= \
        _lib.RA_NOALLOC_SCRATCH_BYTES


def test_microbench_exports_and_validation():
    """The ceiling microbenchmarks' library exports what include/ra_microbench.h
    declares and rejects bad arguments before any HIP call."""
    from paper_2603_18815_amd import microbench as mb
    text = open(os.path.join(ROOT, "include", "ra_microbench.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    declared = set(re.findall(r"^\s*int\s+(\w+)\s*\(", text, flags=re.M))
    assert declared == set(mb.EXPORTS), declared
    lib = mb.load()
    for n in declared:
        assert hasattr(lib, n), n
    assert lib.ra_mb_block_read(None, 1 << 20, 4096, 4, FAKE, None) == 1
    assert lib.ra_mb_block_read(FAKE, 1 << 20, 3000, 4, FAKE, None) == 2   # block size
    assert lib.ra_mb_block_read(FAKE, 3 << 20, 4096, 4, FAKE, None) == 2   # not a power of two
    assert lib.ra_mb_block_read(FAKE, 8 * 4096, 4096, 4, FAKE, None) == 2  # under 16 blocks
    assert lib.ra_mb_block_read(FAKE, 1 << 20, 4096, 0, FAKE, None) == 2
    assert lib.ra_mb_l2_read(None, 1 << 21, 1, 4, 10, FAKE, None) == 1
    assert lib.ra_mb_l2_read(FAKE, 3 << 20, 1, 4, 10, FAKE, None) == 2    # not a power of two
    assert lib.ra_mb_l2_read(FAKE, 1 << 15, 1, 4, 10, FAKE, None) == 2    # under 64 KiB
    assert lib.ra_mb_l2_read(FAKE, 1 << 21, 0, 4, 0, FAKE, None) == 2     # no rounds
    assert lib.ra_mb_l2_read(FAKE, 1 << 21, 0, 4, 1 << 25, FAKE, None) == 2
    assert lib.ra_mb_stream_read(FAKE, 4095, None, 4, FAKE, None) == 2
    assert lib.ra_mb_stream_read(None, 4096, None, 4, FAKE, None) == 1
    assert lib.ra_mb_mfma_bf16(None, 1, 1, FAKE, FAKE, None) == 1
    assert lib.ra_mb_mfma_bf16(FAKE, 0, 1, FAKE, FAKE, None) == 2
    assert lib.ra_mb_lds_read(1, 0, FAKE, FAKE, None) == 2
