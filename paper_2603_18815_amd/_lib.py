"""ctypes declarations of the C ABI in include/rollout_attn.h (argument marshalling only)."""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librollout_attn.so")

RA_OK = 0
RA_ERR_NULL = 1
RA_ERR_SHAPE = 2
RA_ERR_UNSUPPORTED = 3
RA_ERR_WORKSPACE = 4
RA_ERR_HIP = 5

RA_KV_BF16 = 0
RA_KV_FP8_E4M3 = 1

RA_NOALLOC_SCRATCH_BYTES = 64 << 20

EXPORTS = (
    "ra_abi_version",
    "ra_status_string",
    "rollout_attn_decode_workspace_size",
    "rollout_attn_decode",
    "rollout_attn_decode_noalloc",
    "rollout_attn_decode_shared_prefix_workspace_size",
    "rollout_attn_decode_shared_prefix",
    "rollout_attn_append_workspace_size",
    "rollout_attn_append",
    "rollout_attn_append_write",
    "rollout_attn_append_write_rope",
    "rollout_attn_mixed_workspace_size",
    "rollout_attn_mixed",
    "kv_page_write",
    "kv_page_write_rope",
    "kv_page_gather",
    "token_logprob_workspace_size",
    "token_logprob",
    "token_logprob_packed_weight_size",
    "token_logprob_pack_weight",
    "token_logprob_packed",
)


class RaPagedKV(ctypes.Structure):
    _fields_ = [
        ("k_pool", ctypes.c_void_p),
        ("v_pool", ctypes.c_void_p),
        ("block_table", ctypes.c_void_p),
        ("num_pages", ctypes.c_int32),
        ("bt_stride", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("kv_dtype", ctypes.c_int32),
        ("k_scale", ctypes.c_float),
        ("v_scale", ctypes.c_float),
    ]


class RolloutAttnError(RuntimeError):
    def __init__(self, fn: str, status: int, name: str):
        super().__init__(f"{fn} returned {name} ({status})")
        self.status = status


_lib = None


def load() -> ctypes.CDLL:
    """Load the built library. Raises if it is missing: there is no fallback path."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built; run `python -m paper_2603_18815_amd.build` "
            "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(LIB_PATH)
    i32, vp, sz, f32 = ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_float
    kvp = ctypes.POINTER(RaPagedKV)
    lib.ra_abi_version.argtypes = []
    lib.ra_abi_version.restype = ctypes.c_int
    lib.ra_status_string.argtypes = [ctypes.c_int]
    lib.ra_status_string.restype = ctypes.c_char_p
    lib.rollout_attn_decode_workspace_size.argtypes = [i32, i32, i32, i32]
    lib.rollout_attn_decode_workspace_size.restype = sz
    lib.rollout_attn_decode.argtypes = [vp, kvp, vp, i32, i32, i32, f32, vp, vp, vp, sz, vp]
    lib.rollout_attn_decode.restype = ctypes.c_int
    lib.rollout_attn_decode_noalloc.argtypes = [vp, kvp, vp, i32, i32, i32, f32, vp, vp, vp]
    lib.rollout_attn_decode_noalloc.restype = ctypes.c_int
    lib.rollout_attn_decode_shared_prefix_workspace_size.argtypes = [i32, i32, i32, i32, i32]
    lib.rollout_attn_decode_shared_prefix_workspace_size.restype = sz
    lib.rollout_attn_decode_shared_prefix.argtypes = [vp, kvp, vp, vp, vp, i32, i32, i32, i32,
                                                      i32, i32, f32, vp, vp, vp, sz, vp]
    lib.rollout_attn_decode_shared_prefix.restype = ctypes.c_int
    lib.rollout_attn_append_workspace_size.argtypes = [i32, i32, i32, i32]
    lib.rollout_attn_append_workspace_size.restype = sz
    lib.rollout_attn_append.argtypes = [vp, vp, vp, kvp, i32, i32, i32, i32, i32, f32, vp, vp,
                                        vp, sz, vp]
    lib.rollout_attn_append.restype = ctypes.c_int
    lib.rollout_attn_append_write.argtypes = [vp, vp, vp, vp, vp, kvp, i32, i32, i32, i32, i32,
                                              f32, vp, vp, vp, sz, vp]
    lib.rollout_attn_append_write.restype = ctypes.c_int
    lib.rollout_attn_append_write_rope.argtypes = [vp, vp, vp, vp, vp, kvp, i32, i32, i32, i32,
                                                   i32, f32, vp, i32, vp, vp, vp, sz, vp]
    lib.rollout_attn_append_write_rope.restype = ctypes.c_int
    lib.rollout_attn_mixed_workspace_size.argtypes = [i32, i32, i32, i32, i32, i32, i32]
    lib.rollout_attn_mixed_workspace_size.restype = sz
    lib.rollout_attn_mixed.argtypes = [vp, kvp, vp, i32, i32, vp, vp,
                                       vp, vp, vp, kvp, i32, i32, i32, i32, vp, vp,
                                       i32, f32, vp, sz, vp]
    lib.rollout_attn_mixed.restype = ctypes.c_int
    lib.token_logprob_workspace_size.argtypes = [i32, i32, i32]
    lib.token_logprob_workspace_size.restype = sz
    lib.token_logprob.argtypes = [vp, vp, vp, i32, i32, i32, f32, vp, vp, vp, sz, vp]
    lib.token_logprob.restype = ctypes.c_int
    lib.token_logprob_packed_weight_size.argtypes = [i32, i32]
    lib.token_logprob_packed_weight_size.restype = sz
    lib.token_logprob_pack_weight.argtypes = [vp, i32, i32, vp, sz, vp]
    lib.token_logprob_pack_weight.restype = ctypes.c_int
    lib.token_logprob_packed.argtypes = [vp, vp, vp, i32, i32, i32, f32, vp, vp, vp, sz, vp]
    lib.token_logprob_packed.restype = ctypes.c_int
    lib.kv_page_write.argtypes = [vp, vp, vp, vp, kvp, i32, i32, i32, i32, vp]
    lib.kv_page_write.restype = ctypes.c_int
    lib.kv_page_write_rope.argtypes = [vp, vp, vp, vp, kvp, i32, i32, i32, i32, vp, i32, vp]
    lib.kv_page_write_rope.restype = ctypes.c_int
    lib.kv_page_gather.argtypes = [kvp, vp, vp, i32, i32, i32, vp, vp, vp]
    lib.kv_page_gather.restype = ctypes.c_int
    _lib = lib
    return lib


def check(fn: str, status: int) -> None:
    if status != RA_OK:
        raise RolloutAttnError(fn, status, load().ra_status_string(status).decode())
