"""The C-ABI library loads and exports every symbol include/mvk.h declares;
host-side argument checks (no device work is enqueued on these paths)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mvk.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mvk_[a-z0-9_]+)\s*\(", text)))


def _lib():
    from paper_2609_10264_amd import _lib as L
    if not os.path.exists(L.LIB_PATH):
        pytest.skip("libmvk.so not built (run __graft_entry__.build())")
    return L


def test_header_declares_expected_calls():
    names = _declared()
    for fn in ("mvk_server_eval", "mvk_keygen", "mvk_encode", "mvk_decode_verify"):
        assert fn in names


def test_library_exports_every_declared_symbol():
    L = _lib()
    lib = ctypes.CDLL(L.LIB_PATH)
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing
    assert sorted(L.EXPORTS) == _declared()


def test_both_field_builds_load_and_export_every_symbol():
    L = _lib()
    for p, path in L.LIB_PATHS.items():
        if not os.path.exists(path):
            pytest.skip(f"{os.path.basename(path)} not built")
        raw = ctypes.CDLL(path)
        assert not [n for n in _declared() if not hasattr(raw, n)]
        lib = L.load(p)
        assert lib.mvk_field_modulus() == p and lib.mvk_abi_version() == L.ABI_VERSION
    assert sorted(L.LIB_PATHS) == [L.MVK_PRIME_BABYBEAR, L.MVK_PRIME] == [15 * 2**27 + 1, 2**31 - 1]
    with pytest.raises(ValueError):
        L.load(97)


def test_abi_version_and_status_strings():
    L = _lib()
    lib = L.load()
    assert lib.mvk_abi_version() == L.ABI_VERSION
    assert lib.mvk_status_str(0) == b"ok"
    assert lib.mvk_status_str(L.MVK_ERANGE) == b"size or value out of range"
    assert lib.mvk_status_str(12345) == b"unknown status"


def test_struct_layouts_match_header():
    L = _lib()
    # two uint32 then four pointers
    assert ctypes.sizeof(L.MvkCode) == 8 + 4 * 8
    assert ctypes.sizeof(L.MvkKey) == 8 + 2 * ctypes.sizeof(L.MvkCode) + 16
    assert ctypes.sizeof(L.MvkSparse) == 16 + 8


def test_host_argument_checks_without_device_work():
    L = _lib()
    lib = L.load()
    fake = ctypes.c_void_p(0x1000)
    # empty problems are no-ops
    assert lib.mvk_server_eval(None, 0, 16, None, 1, None, None) == L.MVK_OK
    assert lib.mvk_server_eval(None, 16, 16, None, 0, None, None) == L.MVK_OK
    # missing output
    assert lib.mvk_server_eval(fake, 4, 16, fake, 1, None, None) == L.MVK_EINVAL
    # n beyond the int32 exactness bound of the limb accumulation
    assert lib.mvk_server_eval(fake, 4, L.MVK_MAX_N + 1, fake, 1, fake, None) == L.MVK_ERANGE
    # inconsistent key: code dimension must equal n / m
    code = L.MvkCode(5, 3, 0x1000, 0x1000, 0x1000, 0x1000)
    key = L.MvkKey(8, 8, code, code, 0x1000, 0x1000)
    assert lib.mvk_keygen(ctypes.byref(key), fake, None) == L.MVK_EINVAL
    assert lib.mvk_keygen(None, fake, None) == L.MVK_EINVAL
    bad = L.MvkCode(8, 0, 0x1000, 0x1000, 0x1000, 0x1000)
    assert lib.mvk_raa_encode(ctypes.byref(bad), fake, 1, fake, None) == L.MVK_EINVAL
    nullcode = L.MvkCode(8, 2, 0, 0x1000, 0x1000, 0x1000)
    assert lib.mvk_raa_syndrome(ctypes.byref(nullcode), fake, 1, fake, None) == L.MVK_EINVAL
    # compute-unit streams: an empty range or no output pointer
    h = ctypes.c_void_p()
    assert lib.mvk_stream_create_cu_range(0, 0, ctypes.byref(h)) == L.MVK_EINVAL
    assert lib.mvk_stream_create_cu_range(0, 8, None) == L.MVK_EINVAL
    assert lib.mvk_stream_destroy(None) == L.MVK_EINVAL


def test_sizes_no_buffer_can_hold_are_rejected():
    """Sizes whose buffers would exceed 2^62 bytes, and vector counts beyond the
    syndrome kernels' grid dimension, return MVK_ERANGE before any device work."""
    L = _lib()
    lib = L.load()
    fake = ctypes.c_void_p(0x1000)
    # keygen: Nx * m words of scratch with Nx = 2^31 - 1, m = 2^31 - 1
    cx = L.MvkCode(1, 0x7FFFFFFF, 0x1000, 0x1000, 0x1000, 0x1000)
    cy = L.MvkCode(0x7FFFFFFF, 1, 0x1000, 0x1000, 0x1000, 0x1000)
    key = L.MvkKey(0x7FFFFFFF, 1, cx, cy, 0x1000, 0x1000)
    assert lib.mvk_keygen(ctypes.byref(key), fake, None) == L.MVK_ERANGE
    # raa_encode: N * count words of scratch
    big = L.MvkCode(1 << 30, 1, 0x1000, 0x1000, 0x1000, 0x1000)
    assert lib.mvk_raa_encode(ctypes.byref(big), fake, 0xFFFFFFFF, fake, None) == L.MVK_ERANGE
    # syndromes of more than 65535 vectors in one call
    small = L.MvkCode(8, 2, 0x1000, 0x1000, 0x1000, 0x1000)
    assert lib.mvk_raa_syndrome(ctypes.byref(small), fake, 65536, fake, None) == L.MVK_ERANGE
    key8 = L.MvkKey(8, 8, small, small, 0x1000, 0x1000)
    ex = L.MvkSparse(None, None, 0, 65536)
    assert lib.mvk_encode(ctypes.byref(key8), fake, 65536, ctypes.byref(ex), fake, None) == L.MVK_ERANGE
    # batch_preprocess: N * N' words of scratch
    qs = (ctypes.c_void_p * 1)(0x1000)
    c2 = L.MvkCode(1 << 30, 1, 0x1000, 0x1000, 0x1000, 0x1000)
    assert lib.mvk_batch_preprocess(1, qs, 0xFFFFFFFF, 1 << 30, ctypes.byref(c2), fake, fake, None) == L.MVK_ERANGE


def test_verify_argument_checks_without_device_work():
    L = _lib()
    lib = L.load()
    fake = ctypes.c_void_p(0x1000)
    code = L.MvkCode(8, 3, 0x1000, 0x1000, 0x1000, 0x1000)
    key = L.MvkKey(8, 8, code, code, 0x1000, 0x1000)
    ex = L.MvkSparse(0x1000, 0x1000, 2, 1)
    too_many = L.MvkSparse(0x1000, 0x1000, 2, 17)  # more than 16 repetitions
    none = L.MvkSparse(0x1000, 0x1000, 2, 0)
    too_long = L.MvkSparse(0x1000, 0x1000, 25, 2)  # t_y > Ny = 24
    for ey, want in ((too_many, L.MVK_ERANGE), (none, L.MVK_EINVAL), (too_long, L.MVK_EINVAL)):
        assert lib.mvk_verify_prepare(ctypes.byref(key), ctypes.byref(ey), fake, None) == want
        assert lib.mvk_decode_verify(ctypes.byref(key), fake, fake, 1, ctypes.byref(ex), ctypes.byref(ey),
                                     fake, None, None, fake, None) == want
        assert lib.mvk_decode_verify_prepared(ctypes.byref(key), fake, fake, 1, ctypes.byref(ex),
                                              ctypes.byref(ey), fake, fake, None, None, fake, None) == want
    ey = L.MvkSparse(0x1000, 0x1000, 2, 2)
    assert lib.mvk_verify_prepare(ctypes.byref(key), ctypes.byref(ey), None, None) == L.MVK_EINVAL
    assert lib.mvk_decode_verify_prepared(ctypes.byref(key), fake, fake, 1, ctypes.byref(ex), ctypes.byref(ey),
                                          None, fake, None, None, fake, None) == L.MVK_EINVAL
    # noise of the wrong column count
    ex3 = L.MvkSparse(0x1000, 0x1000, 2, 3)
    assert lib.mvk_decode_verify(ctypes.byref(key), fake, fake, 1, ctypes.byref(ex3), ctypes.byref(ey),
                                 fake, None, None, fake, None) == L.MVK_EINVAL


def test_packed_weight_size_and_checks():
    L = _lib()
    lib = L.load()
    assert lib.mvk_packed_weight_bytes(0, 5) == 0 and lib.mvk_packed_weight_bytes(5, 0) == 0
    assert lib.mvk_packed_weight_bytes(1, 1) == 1024
    assert lib.mvk_packed_weight_bytes(17, 65) == 2 * 2 * 1024
    assert lib.mvk_packed_weight_bytes(28672, 8192) == 28672 * 8192
    fake = ctypes.c_void_p(0x1000)
    odd = ctypes.c_void_p(0x1001)
    assert lib.mvk_pack_weights(fake, 0, 4, None, None) == L.MVK_OK
    assert lib.mvk_pack_weights(fake, 4, 4, None, None) == L.MVK_EINVAL
    assert lib.mvk_pack_weights(fake, 4, 4, odd, None) == L.MVK_EINVAL
    assert lib.mvk_server_eval_packed(odd, 4, 16, fake, 1, fake, None) == L.MVK_EINVAL
    assert lib.mvk_server_eval_packed(fake, 4, L.MVK_MAX_N + 1, fake, 1, fake, None) == L.MVK_ERANGE
    assert lib.mvk_server_eval_packed(fake, 0, 16, fake, 1, fake, None) == L.MVK_OK


def test_prepared_path_argument_checks_without_device_work():
    L = _lib()
    lib = L.load()
    fake = ctypes.c_void_p(0x1000)
    code = L.MvkCode(8, 3, 0x1000, 0x1000, 0x1000, 0x1000)
    key = L.MvkKey(8, 8, code, code, 0x1000, 0x1000)
    ex = L.MvkSparse(0x1000, 0x1000, 2, 1)
    ey = L.MvkSparse(0x1000, 0x1000, 2, 2)
    def prep(*a):
        return lib.mvk_client_prepare(*a[:7], None, 0, a[7])

    # nothing to prepare
    assert prep(ctypes.byref(key), None, None, None, None, None, None, None) == L.MVK_OK
    # a done flag needs a nonzero value
    assert lib.mvk_client_prepare(ctypes.byref(key), None, None, None, None, None, None, fake, 0,
                                  None) == L.MVK_EINVAL
    # masks requested without their outputs
    assert prep(ctypes.byref(key), ctypes.byref(ex), None, None, fake, None, None, None) == L.MVK_EINVAL
    assert prep(ctypes.byref(key), ctypes.byref(ex), None, fake, None, None, None, None) == L.MVK_EINVAL
    # noise longer than Nx = 24; too many noise vectors
    assert prep(ctypes.byref(key), ctypes.byref(L.MvkSparse(0x1000, 0x1000, 25, 1)), None, fake, fake, None,
                None, None) == L.MVK_EINVAL
    assert prep(ctypes.byref(key), ctypes.byref(L.MvkSparse(0x1000, 0x1000, 2, 65536)), None, fake, fake, None,
                None, None) == L.MVK_ERANGE
    # challenges: the checks of verify, and both outputs required
    assert prep(ctypes.byref(key), None, ctypes.byref(L.MvkSparse(0x1000, 0x1000, 2, 17)), None, None, fake,
                fake, None) == L.MVK_ERANGE
    assert prep(ctypes.byref(key), None, ctypes.byref(ey), None, None, fake, None, None) == L.MVK_EINVAL
    assert prep(ctypes.byref(key), None, ctypes.byref(ey), None, None, None, fake, None) == L.MVK_EINVAL
    # encode with a prepared mask
    enc = lib.mvk_encode_masked
    assert enc(ctypes.byref(key), fake, 0, None, None, None, 0, 0, None, None) == L.MVK_OK
    assert enc(ctypes.byref(key), fake, 1, None, fake, None, 0, 0, None, None) == L.MVK_EINVAL
    assert enc(ctypes.byref(key), fake, 1, fake, fake, fake, 0, 10, None, None) == L.MVK_EINVAL  # value 0
    assert enc(ctypes.byref(key), fake, 1, fake, fake, fake, 1, 0, None, None) == L.MVK_EINVAL  # no time-out
    # decode/verify with prepared masks: 1 <= ell <= 16, every input present
    dvm = lib.mvk_decode_verify_masked
    assert dvm(ctypes.byref(key), fake, fake, 1, fake, 0, fake, fake, fake, None, None, fake, None) == L.MVK_EINVAL
    assert dvm(ctypes.byref(key), fake, fake, 1, fake, 17, fake, fake, fake, None, None, fake, None) == L.MVK_ERANGE
    assert dvm(ctypes.byref(key), fake, fake, 1, fake, 2, fake, None, fake, None, None, fake, None) == L.MVK_EINVAL
    assert dvm(ctypes.byref(key), fake, fake, 1, None, 2, fake, fake, fake, None, None, fake, None) == L.MVK_EINVAL
    assert dvm(ctypes.byref(key), fake, fake, 0, None, 2, None, None, None, None, None, None, None) == L.MVK_OK
    # stream flags
    assert lib.mvk_flag_signal(None, 1, None) == L.MVK_EINVAL
    assert lib.mvk_flag_signal(fake, 0, None) == L.MVK_EINVAL
    assert lib.mvk_flag_wait(None, 1, 10, None, None) == L.MVK_EINVAL
    assert lib.mvk_flag_wait(fake, 0, 10, None, None) == L.MVK_EINVAL
    assert lib.mvk_flag_wait(fake, 1, 0, None, None) == L.MVK_EINVAL


def test_verify_only_argument_checks_without_device_work():
    L = _lib()
    lib = L.load()
    fake = ctypes.c_void_p(0x1000)
    code = L.MvkCode(8, 3, 0x1000, 0x1000, 0x1000, 0x1000)
    key = L.MvkKey(8, 8, code, code, 0x1000, 0x1000)
    ey = L.MvkSparse(0x1000, 0x1000, 2, 2)
    assert lib.mvk_verify(ctypes.byref(key), fake, fake, 0, ctypes.byref(ey), None, None, None, None) == L.MVK_OK
    assert lib.mvk_verify(ctypes.byref(key), None, fake, 1, ctypes.byref(ey), None, None, fake, None) == L.MVK_EINVAL
    assert lib.mvk_verify(ctypes.byref(key), fake, fake, 1, ctypes.byref(ey), None, None, None, None) == L.MVK_EINVAL
    assert lib.mvk_verify(ctypes.byref(key), fake, fake, 1, ctypes.byref(L.MvkSparse(0x1000, 0x1000, 2, 17)),
                          None, None, fake, None) == L.MVK_ERANGE
    assert lib.mvk_verify(ctypes.byref(key), fake, fake, 1, ctypes.byref(L.MvkSparse(0x1000, 0x1000, 25, 2)),
                          None, None, fake, None) == L.MVK_EINVAL
    noq = L.MvkKey(8, 8, code, code, 0x1000, 0)
    assert lib.mvk_verify(ctypes.byref(noq), fake, fake, 1, ctypes.byref(ey), None, None, fake, None) == L.MVK_EINVAL


def test_batch_argument_checks_without_device_work():
    L = _lib()
    lib = L.load()
    fake = ctypes.c_void_p(0x1000)
    cy = L.MvkCode(8, 3, 0x1000, 0x1000, 0x1000, 0x1000)   # k = m = 8, N = 24
    c2 = L.MvkCode(12, 2, 0x1000, 0x1000, 0x1000, 0x1000)  # k = B*n = 12, N' = 24
    ptrs = (ctypes.c_void_p * 3)(0x1000, 0x1000, 0x1000)
    pre = lib.mvk_batch_preprocess
    assert pre(0, ptrs, 24, 4, ctypes.byref(c2), fake, fake, None) == L.MVK_EINVAL
    assert pre(3, ptrs, 24, 5, ctypes.byref(c2), fake, fake, None) == L.MVK_EINVAL  # c2.k != B*n
    assert pre(3, ptrs, 24, 4, ctypes.byref(c2), None, fake, None) == L.MVK_EINVAL
    nulls = (ctypes.c_void_p * 3)(0x1000, 0, 0x1000)
    assert pre(3, nulls, 24, 4, ctypes.byref(c2), fake, fake, None) == L.MVK_EINVAL
    e = L.MvkSparse(0x1000, 0x1000, 2, 2)
    assert lib.mvk_batch_project(fake, 24, 4, 3, ctypes.byref(L.MvkSparse(0x1000, 0x1000, 2, 17)), fake,
                                 None) == L.MVK_ERANGE
    assert lib.mvk_batch_project(fake, 24, 4, 3, ctypes.byref(L.MvkSparse(0x1000, 0x1000, 25, 2)), fake,
                                 None) == L.MVK_EINVAL
    assert lib.mvk_batch_project(fake, 24, 4, 3, ctypes.byref(e), None, None) == L.MVK_EINVAL
    ver = lib.mvk_batch_verify
    args = lambda **kw: dict(dict(cy=ctypes.byref(cy), c2=ctypes.byref(c2), Qaux=fake, m=8, n=4, B=3, X=fake,  # noqa: E731
                                  Y=fake, e=ctypes.byref(e), Ut=fake, e2=ctypes.byref(e), acc=fake), **kw)

    def call(a):
        return ver(a["cy"], a["c2"], a["Qaux"], a["m"], a["n"], a["B"], a["X"], a["Y"], a["e"], a["Ut"], a["e2"],
                   None, None, None, None, a["acc"], None)

    assert call(args(B=0)) == L.MVK_OK
    assert call(args(n=5)) == L.MVK_EINVAL               # secondary code dimension != B*n
    assert call(args(m=9)) == L.MVK_EINVAL               # primary code dimension != m
    assert call(args(acc=None)) == L.MVK_EINVAL
    assert call(args(e2=ctypes.byref(L.MvkSparse(0x1000, 0x1000, 2, 17)))) == L.MVK_ERANGE
    assert call(args(e2=ctypes.byref(L.MvkSparse(0x1000, 0x1000, 25, 2)))) == L.MVK_EINVAL  # t' > N' = 24
    assert call(args(e=ctypes.byref(L.MvkSparse(0x1000, 0x1000, 25, 2)))) == L.MVK_EINVAL   # t > N = 24


def test_stream_read_argument_checks_without_device_work():
    L = _lib()
    lib = L.load()
    fake = ctypes.c_void_p(0x1000)
    assert lib.mvk_stream_read(None, 0, None, None) == L.MVK_OK  # empty read
    assert lib.mvk_stream_read(None, 64, fake, None) == L.MVK_EINVAL
    assert lib.mvk_stream_read(fake, 64, None, None) == L.MVK_EINVAL
    assert lib.mvk_stream_read(ctypes.c_void_p(0x1004), 64, fake, None) == L.MVK_EINVAL  # misaligned
    assert lib.mvk_stream_read(fake, 60, fake, None) == L.MVK_EINVAL  # not a multiple of 16


def test_seeded_call_argument_checks_without_device_work():
    """The seeded calls reject bad sizes and pointers before any allocation or
    launch; the accessors and frees accept NULL."""
    L = _lib()
    lib = L.load()
    fake = ctypes.c_void_p(0x1000)
    out = ctypes.c_void_p()
    assert lib.mvk_keygen_seeded(8, 8, 3, 3, 1, None, None, ctypes.byref(out)) == L.MVK_EINVAL
    assert lib.mvk_keygen_seeded(8, 8, 3, 3, 1, fake, None, None) == L.MVK_EINVAL
    assert lib.mvk_keygen_seeded(8, 8, 0, 3, 1, fake, None, ctypes.byref(out)) == L.MVK_EINVAL
    assert lib.mvk_keygen_seeded(8, L.MVK_MAX_N + 1, 3, 3, 1, fake, None, ctypes.byref(out)) == L.MVK_ERANGE
    assert lib.mvk_keygen_seeded(1 << 30, 8, 3, 3, 1, fake, None, ctypes.byref(out)) == L.MVK_ERANGE  # Ny > 2^31-1
    assert out.value is None
    code = L.MvkCode(8, 2, 0x1000, 0x1000, 0x1000, 0x1000)
    key = L.MvkKey(8, 8, code, code, 0x1000, 0x1000)
    st = ctypes.c_void_p()
    assert lib.mvk_encode_seeded(ctypes.byref(key), fake, 2, 4, 1, fake, None, None) == L.MVK_EINVAL
    assert lib.mvk_encode_seeded(ctypes.byref(key), fake, 2, 17, 1, fake, ctypes.byref(st), None) == L.MVK_EINVAL
    assert lib.mvk_encode_seeded(ctypes.byref(key), fake, 2, L.MVK_SEEDED_MAX_T + 1, 1, fake, ctypes.byref(st),
                                 None) == L.MVK_ERANGE
    assert lib.mvk_encode_seeded(ctypes.byref(key), fake, 65536, 4, 1, fake, ctypes.byref(st), None) == L.MVK_ERANGE
    assert lib.mvk_encode_seeded(ctypes.byref(key), None, 2, 4, 1, fake, ctypes.byref(st), None) == L.MVK_EINVAL
    assert st.value is None
    assert lib.mvk_decode_verify_seeded(ctypes.byref(key), None, fake, fake, 4, 2, 1, fake, None, None, fake,
                                        None) == L.MVK_EINVAL
    assert not lib.mvk_pp_key(None)
    assert lib.mvk_st_noise(None) is not None and not lib.mvk_st_noise(None)
    lib.mvk_pp_free(None)
    lib.mvk_st_free(None)
    assert lib.mvk_status_str(L.MVK_ERANDOM) != b"unknown status"
    assert lib.mvk_status_str(L.MVK_ECAPTURE) != b"unknown status"


def test_static_server_eval_rejects_shapes_beyond_its_scratch():
    """mvk_server_eval_packed_static checks the shape's scratch against its
    static array on the host, before any device work: 28672 x 131071 with 64
    queries needs 46 MiB of split-k partial sums and digit tiles (limit
    MVK_STATIC_SCRATCH_BYTES = 32 MiB)."""
    L = _lib()
    lib = L.load()
    fake = ctypes.c_void_p(0x1000)
    assert L.MVK_STATIC_SCRATCH_BYTES == 32 << 20
    assert lib.mvk_server_eval_packed_static(fake, 28672, 131071, fake, 64, fake, None) == L.MVK_ERANGE
    assert lib.mvk_server_eval_packed_static(fake, 4, L.MVK_MAX_N + 1, fake, 1, fake, None) == L.MVK_ERANGE
    assert lib.mvk_server_eval_packed_static(ctypes.c_void_p(0x1001), 4, 16, fake, 1, fake, None) == L.MVK_EINVAL
    assert lib.mvk_server_eval_packed_static(fake, 4, 16, fake, 1, None, None) == L.MVK_EINVAL
    assert lib.mvk_server_eval_packed_static(None, 0, 16, None, 1, None, None) == L.MVK_OK
    # row or query counts whose rounded-up tile counts would wrap in 32 bits
    assert lib.mvk_server_eval_packed_static(fake, 0xFFFFFFFF, 131071, fake, 0xFFFFFFFF, fake, None) == L.MVK_ERANGE
    assert lib.mvk_server_eval_packed_static(fake, 0xFFFFFFF0, 64, fake, 64, fake, None) == L.MVK_ERANGE
    assert lib.mvk_server_eval(fake, 0xFFFFFFF0, 64, fake, 1, fake, None) == L.MVK_ERANGE
    assert lib.mvk_server_eval_packed(fake, 16, 64, fake, 0x80000000, fake, None) == L.MVK_ERANGE
    assert lib.mvk_pack_weights(fake, 0xFFFFFFF0, 64, fake, None) == L.MVK_ERANGE


def test_group_server_eval_argument_checks_without_device_work():
    L = _lib()
    lib = L.load()
    fake = ctypes.c_void_p(0x1000)
    ys = (ctypes.c_void_p * 4)(0x1000, 0x1000, 0x1000, 0x1000)
    assert L.MVK_MAX_GROUP == 4
    assert lib.mvk_server_eval_packed_group(fake, 0, 16, 64, fake, 1, ys, None) == L.MVK_EINVAL
    assert lib.mvk_server_eval_packed_group(fake, 5, 16, 64, fake, 1, ys, None) == L.MVK_EINVAL
    assert lib.mvk_server_eval_packed_group(fake, 2, 17, 64, fake, 1, ys, None) == L.MVK_EINVAL  # m % 16
    assert lib.mvk_server_eval_packed_group(fake, 2, 16, 64, fake, 1, None, None) == L.MVK_EINVAL
    nully = (ctypes.c_void_p * 2)(0x1000, None)
    assert lib.mvk_server_eval_packed_group(fake, 2, 16, 64, fake, 1, nully, None) == L.MVK_EINVAL
    assert lib.mvk_server_eval_packed_group(fake, 4, 0x40000000, 64, fake, 1, ys, None) == L.MVK_ERANGE
    assert lib.mvk_server_eval_packed_group(fake, 2, 16, L.MVK_MAX_N + 1, fake, 1, ys, None) == L.MVK_ERANGE
    assert lib.mvk_server_eval_packed_group(ctypes.c_void_p(0x1008), 2, 16, 64, fake, 1, ys, None) == L.MVK_EINVAL
    assert lib.mvk_server_eval_packed_group(fake, 2, 0, 64, fake, 1, ys, None) == L.MVK_OK
