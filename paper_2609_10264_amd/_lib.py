"""ctypes loader and C struct layouts for the libraries behind include/mvk.h:
libmvk.so (p = 2^31 - 1) and libmvk_bb.so (BabyBear, p = 15 * 2^27 + 1)."""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmvk.so")
LIB_PATH_BB = os.path.join(_HERE, "libmvk_bb.so")

MVK_OK = 0
MVK_EINVAL = -1
MVK_ERANGE = -2
MVK_ENOMEM = -3
MVK_EHIP = -4
MVK_ERANDOM = -5
MVK_ECAPTURE = -6
MVK_PRIME = 2147483647
MVK_PRIME_BABYBEAR = 2013265921
MVK_MAX_N = 131071
MVK_PATH_AUTO = 0
MVK_PATH_VALU = 1
MVK_PATH_MFMA = 2
MVK_STREAM_READ_BLOCKS = 4096
MVK_TAG_CODE_X = 0x6D766B2D636F6478
MVK_TAG_CODE_Y = 0x6D766B2D636F6479
MVK_TAG_NOISE = 0x6D766B2D6E6F6973
MVK_TAG_CHALLENGE = 0x6D766B2D6368616C
MVK_SEED_FRESH = 0xFFFFFFFFFFFFFFFF
MVK_SEEDED_MAX_T = 4096
MVK_STATIC_SCRATCH_BYTES = 32 << 20
MVK_MAX_GROUP = 4
MVK_MAX_PREP = 8
ABI_VERSION = 9
# field modulus -> library built over that field
LIB_PATHS = {MVK_PRIME: LIB_PATH, MVK_PRIME_BABYBEAR: LIB_PATH_BB}

# Every symbol include/mvk.h declares.
EXPORTS = (
    "mvk_status_str",
    "mvk_abi_version",
    "mvk_field_modulus",
    "mvk_server_eval",
    "mvk_server_eval_path",
    "mvk_packed_weight_bytes",
    "mvk_pack_weights",
    "mvk_server_eval_packed",
    "mvk_keygen",
    "mvk_encode",
    "mvk_decode_verify",
    "mvk_verify",
    "mvk_verify_prepare",
    "mvk_decode_verify_prepared",
    "mvk_client_prepare",
    "mvk_encode_masked",
    "mvk_decode_verify_masked",
    "mvk_flag_signal",
    "mvk_flag_wait",
    "mvk_batch_preprocess",
    "mvk_batch_project",
    "mvk_batch_verify",
    "mvk_raa_encode",
    "mvk_raa_syndrome",
    "mvk_stream_read",
    "mvk_workspace_release",
    "mvk_sample_code",
    "mvk_sample_sparse",
    "mvk_keygen_seeded",
    "mvk_pp_key",
    "mvk_pp_free",
    "mvk_encode_seeded",
    "mvk_st_noise",
    "mvk_st_free",
    "mvk_decode_verify_seeded",
    "mvk_server_eval_packed_static",
    "mvk_server_eval_packed_group",
    "mvk_decode_verify_masked_group",
    "mvk_client_prepare_group",
    "mvk_client_prepare_multi",
    "mvk_stream_create_cu_range",
    "mvk_stream_destroy",
    "mvk_decode_verify_encode_masked",
)


class MvkCode(ctypes.Structure):
    _fields_ = [
        ("k", ctypes.c_uint32),
        ("r", ctypes.c_uint32),
        ("pi1", ctypes.c_void_p),
        ("pi2", ctypes.c_void_p),
        ("v1", ctypes.c_void_p),
        ("v2", ctypes.c_void_p),
    ]


class MvkKey(ctypes.Structure):
    _fields_ = [
        ("m", ctypes.c_uint32),
        ("n", ctypes.c_uint32),
        ("cx", MvkCode),
        ("cy", MvkCode),
        ("PT", ctypes.c_void_p),
        ("Q", ctypes.c_void_p),
    ]


class MvkSparse(ctypes.Structure):
    _fields_ = [
        ("idx", ctypes.c_void_p),
        ("val", ctypes.c_void_p),
        ("t", ctypes.c_uint32),
        ("count", ctypes.c_uint32),
    ]


class MvkError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn} failed: {msg} (status {status})")
        self.status = status


_libs: dict = {}


def load(p: int = MVK_PRIME) -> ctypes.CDLL:
    """Load the library built over F_p; raises if it has not been built."""
    L = _libs.get(p)
    if L is not None:
        return L
    if p not in LIB_PATHS:
        raise ValueError(f"no build over p = {p}; fields: {sorted(LIB_PATHS)}")
    path = LIB_PATHS[p]
    if not os.path.exists(path):
        raise ImportError(f"{path} not found: build it with `python -m paper_2609_10264_amd.build` "
                          "(there is no fallback implementation)")
    L = ctypes.CDLL(path)
    st = ctypes.c_int32
    vp = ctypes.c_void_p
    u32 = ctypes.c_uint32
    L.mvk_status_str.argtypes = [st]
    L.mvk_status_str.restype = ctypes.c_char_p
    L.mvk_abi_version.argtypes = []
    L.mvk_abi_version.restype = ctypes.c_int32
    L.mvk_field_modulus.argtypes = []
    L.mvk_field_modulus.restype = ctypes.c_uint32
    L.mvk_server_eval.argtypes = [vp, u32, u32, vp, u32, vp, vp]
    L.mvk_server_eval.restype = st
    L.mvk_server_eval_path.argtypes = [vp, u32, u32, vp, u32, vp, ctypes.c_int32, vp]
    L.mvk_server_eval_path.restype = st
    L.mvk_packed_weight_bytes.argtypes = [u32, u32]
    L.mvk_packed_weight_bytes.restype = ctypes.c_size_t
    L.mvk_pack_weights.argtypes = [vp, u32, u32, vp, vp]
    L.mvk_pack_weights.restype = st
    L.mvk_server_eval_packed.argtypes = [vp, u32, u32, vp, u32, vp, vp]
    L.mvk_server_eval_packed.restype = st
    L.mvk_keygen.argtypes = [ctypes.POINTER(MvkKey), vp, vp]
    L.mvk_keygen.restype = st
    L.mvk_encode.argtypes = [ctypes.POINTER(MvkKey), vp, u32, ctypes.POINTER(MvkSparse), vp, vp]
    L.mvk_encode.restype = st
    L.mvk_decode_verify.argtypes = [ctypes.POINTER(MvkKey), vp, vp, u32, ctypes.POINTER(MvkSparse),
                                    ctypes.POINTER(MvkSparse), vp, vp, vp, vp, vp]
    L.mvk_decode_verify.restype = st
    L.mvk_verify.argtypes = [ctypes.POINTER(MvkKey), vp, vp, u32, ctypes.POINTER(MvkSparse), vp, vp, vp, vp]
    L.mvk_verify.restype = st
    L.mvk_verify_prepare.argtypes = [ctypes.POINTER(MvkKey), ctypes.POINTER(MvkSparse), vp, vp]
    L.mvk_verify_prepare.restype = st
    L.mvk_decode_verify_prepared.argtypes = [ctypes.POINTER(MvkKey), vp, vp, u32, ctypes.POINTER(MvkSparse),
                                             ctypes.POINTER(MvkSparse), vp, vp, vp, vp, vp, vp]
    L.mvk_decode_verify_prepared.restype = st
    L.mvk_client_prepare.argtypes = [ctypes.POINTER(MvkKey), ctypes.POINTER(MvkSparse), ctypes.POINTER(MvkSparse),
                                     vp, vp, vp, vp, vp, u32, vp]
    L.mvk_client_prepare.restype = st
    L.mvk_encode_masked.argtypes = [ctypes.POINTER(MvkKey), vp, u32, vp, vp, vp, u32, u32, vp, vp]
    L.mvk_encode_masked.restype = st
    L.mvk_decode_verify_masked.argtypes = [ctypes.POINTER(MvkKey), vp, vp, u32, vp, u32, vp, vp, vp, vp, vp, vp, vp]
    L.mvk_decode_verify_masked.restype = st
    L.mvk_flag_signal.argtypes = [vp, u32, vp]
    L.mvk_flag_signal.restype = st
    L.mvk_flag_wait.argtypes = [vp, u32, u32, vp, vp]
    L.mvk_flag_wait.restype = st
    L.mvk_batch_preprocess.argtypes = [u32, ctypes.POINTER(vp), u32, u32, ctypes.POINTER(MvkCode), vp, vp, vp]
    L.mvk_batch_preprocess.restype = st
    L.mvk_batch_project.argtypes = [vp, u32, u32, u32, ctypes.POINTER(MvkSparse), vp, vp]
    L.mvk_batch_project.restype = st
    L.mvk_batch_verify.argtypes = [ctypes.POINTER(MvkCode), ctypes.POINTER(MvkCode), vp, u32, u32, u32, vp, vp,
                                   ctypes.POINTER(MvkSparse), vp, ctypes.POINTER(MvkSparse), vp, vp, vp, vp, vp, vp]
    L.mvk_batch_verify.restype = st
    L.mvk_raa_encode.argtypes = [ctypes.POINTER(MvkCode), vp, u32, vp, vp]
    L.mvk_raa_encode.restype = st
    L.mvk_raa_syndrome.argtypes = [ctypes.POINTER(MvkCode), vp, u32, vp, vp]
    L.mvk_raa_syndrome.restype = st
    L.mvk_stream_read.argtypes = [vp, ctypes.c_size_t, vp, vp]
    L.mvk_stream_read.restype = st
    u64 = ctypes.c_uint64
    u32p = ctypes.POINTER(ctypes.c_uint32)
    L.mvk_workspace_release.argtypes = []
    L.mvk_workspace_release.restype = st
    L.mvk_sample_code.argtypes = [u32, u32, u64, u64, u32p, u32p, u32p, u32p]
    L.mvk_sample_code.restype = st
    L.mvk_sample_sparse.argtypes = [u32, u32, u32, u64, u64, u32p, u32p]
    L.mvk_sample_sparse.restype = st
    L.mvk_keygen_seeded.argtypes = [u32, u32, u32, u32, u64, vp, vp, ctypes.POINTER(vp)]
    L.mvk_keygen_seeded.restype = st
    L.mvk_pp_key.argtypes = [vp]
    L.mvk_pp_key.restype = ctypes.POINTER(MvkKey)
    L.mvk_pp_free.argtypes = [vp]
    L.mvk_pp_free.restype = None
    L.mvk_encode_seeded.argtypes = [ctypes.POINTER(MvkKey), vp, u32, u32, u64, vp, ctypes.POINTER(vp), vp]
    L.mvk_encode_seeded.restype = st
    L.mvk_st_noise.argtypes = [vp]
    L.mvk_st_noise.restype = ctypes.POINTER(MvkSparse)
    L.mvk_st_free.argtypes = [vp]
    L.mvk_st_free.restype = None
    L.mvk_decode_verify_seeded.argtypes = [ctypes.POINTER(MvkKey), vp, vp, vp, u32, u32, u64, vp, vp, vp, vp, vp]
    L.mvk_decode_verify_seeded.restype = st
    L.mvk_server_eval_packed_static.argtypes = [vp, u32, u32, vp, u32, vp, vp]
    L.mvk_server_eval_packed_static.restype = st
    L.mvk_server_eval_packed_group.argtypes = [vp, u32, u32, u32, vp, u32, ctypes.POINTER(vp), vp]
    L.mvk_server_eval_packed_group.restype = st
    pvp = ctypes.POINTER(vp)
    L.mvk_decode_verify_masked_group.argtypes = [u32, ctypes.POINTER(ctypes.POINTER(MvkKey)), vp, u32, pvp, pvp, u32,
                                                 pvp, pvp, pvp, pvp, pvp, pvp, vp]
    L.mvk_decode_verify_masked_group.restype = st
    L.mvk_client_prepare_group.argtypes = [u32, ctypes.POINTER(ctypes.POINTER(MvkKey)), ctypes.POINTER(MvkSparse),
                                           ctypes.POINTER(ctypes.POINTER(MvkSparse)), vp, pvp, pvp, pvp, vp, u32, vp]
    L.mvk_client_prepare_group.restype = st
    L.mvk_client_prepare_multi.argtypes = [u32, ctypes.POINTER(ctypes.POINTER(MvkKey)),
                                           ctypes.POINTER(ctypes.POINTER(MvkSparse)),
                                           ctypes.POINTER(ctypes.POINTER(MvkSparse)), pvp, pvp, pvp, pvp, pvp, u32, vp]
    L.mvk_client_prepare_multi.restype = st
    L.mvk_stream_create_cu_range.argtypes = [u32, u32, ctypes.POINTER(vp)]
    L.mvk_stream_create_cu_range.restype = st
    L.mvk_stream_destroy.argtypes = [vp]
    L.mvk_stream_destroy.restype = st
    L.mvk_decode_verify_encode_masked.argtypes = [ctypes.POINTER(MvkKey), vp, vp, u32, vp, u32, vp, vp, vp, vp, vp,
                                                  vp, vp, u32, vp, vp, vp, u32, u32, vp, vp]
    L.mvk_decode_verify_encode_masked.restype = st
    if L.mvk_abi_version() != ABI_VERSION:
        raise ImportError(f"{path}: ABI version mismatch; rebuild the library")
    if L.mvk_field_modulus() != p:
        raise ImportError(f"{path} is built over p = {L.mvk_field_modulus()}, expected {p}")
    _libs[p] = L
    return L


def check(fn: str, status: int) -> None:
    if status != MVK_OK:
        raise MvkError(fn, status, load().mvk_status_str(status).decode())
