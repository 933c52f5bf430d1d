"""MI355X (gfx950) library for the hot path of private and verifiable
matrix-vector multiplication delegation (pvMVMD, Maverick, arxiv 2609.10264).

Thin Python binding over the C ABI in include/mvk.h: every function only
checks tensor shapes/dtypes, passes raw device pointers and the current HIP
stream, and raises on a non-zero status.  All computation runs in the HIP
kernels of libmvk.so (p = 2^31 - 1) or libmvk_bb.so (BabyBear, p = 15 * 2^27 + 1);
there is no CPU fallback.

Field: every code carries its prime p (P or P_BABYBEAR) and every call runs
in the library built over the p of its codes (or of its `p` argument where no
code is passed).  Tensors: field arrays are torch.int32 on the GPU holding
canonical values in [0, p) (these fit a non-negative int32); W is torch.int8.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass

import torch

from . import _lib
from ._lib import MVK_MAX_N, MVK_PRIME, MVK_PRIME_BABYBEAR, MvkCode, MvkError, MvkKey, MvkSparse

P = MVK_PRIME
P_BABYBEAR = MVK_PRIME_BABYBEAR
FIELDS = {"m31": P, "babybear": P_BABYBEAR}

__all__ = ["P", "P_BABYBEAR", "FIELDS", "MVK_MAX_N", "MvkError", "Code", "Key", "PackedW", "pack_weights", "server_eval",
           "keygen", "encode", "decode_verify", "verify_prepare", "raa_encode", "raa_syndrome", "library_path",
           "keygen_seeded", "encode_seeded", "decode_verify_seeded", "sample_code", "sample_sparse", "SeededPP",
           "SeededState", "TAG_CODE_X", "TAG_CODE_Y", "TAG_NOISE", "TAG_CHALLENGE", "SEED_FRESH"]


def library_path(p: int = P) -> str:
    return _lib.LIB_PATHS[p]


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dev(t: torch.Tensor, dtype: torch.dtype, shape: tuple | None, name: str) -> int:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must have dtype {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t.data_ptr()


@dataclass
class Code:
    """RAA code description (App. B) held on the device: N = r * k."""
    k: int
    r: int
    pi1: torch.Tensor
    pi2: torch.Tensor
    v1: torch.Tensor
    v2: torch.Tensor
    p: int = P  # the field the diagonals (and everything coded with it) live in

    @property
    def N(self) -> int:
        return self.k * self.r

    @classmethod
    def from_arrays(cls, k, r, pi1, pi2, v1, v2, device="cuda", p: int = P) -> "Code":
        def t(a):
            return torch.as_tensor(a).to(torch.int64).to(torch.int32).to(device).contiguous()
        return cls(int(k), int(r), t(pi1), t(pi2), t(v1), t(v2), int(p))

    def struct(self) -> MvkCode:
        N = self.N
        return MvkCode(self.k, self.r,
                       _dev(self.pi1, torch.int32, (N,), "pi1"), _dev(self.pi2, torch.int32, (N,), "pi2"),
                       _dev(self.v1, torch.int32, (N,), "v1"), _dev(self.v2, torch.int32, (N,), "v2"))


@dataclass
class Key:
    """Public parameters pp = (Gx, Gy, P^T, Q) of Protocol pvMVMD."""
    m: int
    n: int
    cx: Code
    cy: Code
    PT: torch.Tensor  # Nx x m
    Q: torch.Tensor   # Ny x n

    @property
    def p(self) -> int:
        return self.cx.p

    @classmethod
    def allocate(cls, m: int, n: int, cx: Code, cy: Code, device="cuda") -> "Key":
        if cx.p != cy.p:
            raise ValueError("the two codes of a key must be over one field")
        PT = torch.empty((cx.N, m), dtype=torch.int32, device=device)
        Q = torch.empty((cy.N, n), dtype=torch.int32, device=device)
        return cls(int(m), int(n), cx, cy, PT, Q)

    def struct(self) -> MvkKey:
        return MvkKey(self.m, self.n, self.cx.struct(), self.cy.struct(),
                      _dev(self.PT, torch.int32, (self.cx.N, self.m), "PT"),
                      _dev(self.Q, torch.int32, (self.cy.N, self.n), "Q"))


def _sparse(idx: torch.Tensor, val: torch.Tensor, name: str) -> MvkSparse:
    if idx.dim() != 2 or idx.shape != val.shape:
        raise ValueError(f"{name}: idx and val must be 2-D of equal shape")
    count, t = idx.shape
    return MvkSparse(_dev(idx, torch.int32, None, name + "_idx"), _dev(val, torch.int32, None, name + "_val"),
                     int(t), int(count))


PATHS = {"auto": _lib.MVK_PATH_AUTO, "valu": _lib.MVK_PATH_VALU, "mfma": _lib.MVK_PATH_MFMA}


class PackedW:
    """W stored in matrix-core operand order (see mvk_pack_weights): a flat int8
    device buffer plus the logical shape m x n."""

    def __init__(self, data: torch.Tensor, m: int, n: int):
        self.data, self.m, self.n = data, m, n

    @property
    def shape(self):
        return (self.m, self.n)

    @property
    def device(self):
        return self.data.device


def pack_weights(W: torch.Tensor, out: torch.Tensor | None = None, stream=None) -> PackedW:
    """Re-lay W (m x n int8, row-major) once into the packed server layout."""
    m, n = W.shape
    L = _lib.load()
    nbytes = int(L.mvk_packed_weight_bytes(m, n))
    if out is None:
        out = torch.empty((max(nbytes, 1),), dtype=torch.int8, device=W.device)
    if out.dtype != torch.int8 or not out.is_contiguous() or out.numel() < nbytes:
        raise ValueError(f"out must be a contiguous int8 buffer of at least {nbytes} bytes")
    _lib.check("mvk_pack_weights", L.mvk_pack_weights(_dev(W, torch.int8, (m, n), "W"), m, n, out.data_ptr(),
                                                      _stream(stream)))
    return PackedW(out, m, n)


def pack_weights_group(Ws: list, stream=None) -> PackedW:
    """The G matrices Ws (each m x n int8, m a multiple of 16 when G > 1) in
    the packed layout of their row stack: G packed buffers back to back."""
    G = len(Ws)
    m, n = Ws[0].shape
    L = _lib.load()
    nbytes = int(L.mvk_packed_weight_bytes(m, n))
    out = torch.empty((max(G * nbytes, 1),), dtype=torch.int8, device=Ws[0].device)
    for g, W in enumerate(Ws):
        if tuple(W.shape) != (m, n):
            raise ValueError("the matrices of a group must have one shape")
        pack_weights(W, out=out[g * nbytes:(g + 1) * nbytes], stream=stream)
    return PackedW(out, G * m, n)


def server_eval_group(Wstack: PackedW, G: int, Xhat: torch.Tensor, outs: list | None = None, stream=None,
                      p: int = P) -> list:
    """[W_g Xhat mod p for g < G] in one launch, Wstack the packed row stack of
    the G matrices (pack_weights_group); returns the G outputs (B x m each)."""
    m = Wstack.m // G
    n = Wstack.n
    B = Xhat.shape[0]
    if outs is None:
        outs = [torch.empty((B, m), dtype=torch.int32, device=Xhat.device) for _ in range(G)]
    ptrs = (ctypes.c_void_p * G)(*[_dev(o, torch.int32, (B, m), f"Yhat[{g}]") for g, o in enumerate(outs)])
    _lib.check("mvk_server_eval_packed_group", _lib.load(p).mvk_server_eval_packed_group(
        Wstack.data.data_ptr(), G, m, n, _dev(Xhat, torch.int32, (B, n), "Xhat"), B, ptrs, _stream(stream)))
    return outs


def server_eval(W, Xhat: torch.Tensor, out: torch.Tensor | None = None, stream=None,
                path: str = "auto", p: int = P) -> torch.Tensor:
    """Yhat = W Xhat mod p.  W: m x n int8 (or a PackedW); Xhat: B x n int32 field; returns B x m.

    path selects the kernel family ("auto", "valu" or "mfma"); results are identical.
    """
    m, n = W.shape
    B = Xhat.shape[0]
    if out is None:
        out = torch.empty((B, m), dtype=torch.int32, device=W.device)
    L = _lib.load(p)
    tail = (m, n, _dev(Xhat, torch.int32, (B, n), "Xhat"), B, _dev(out, torch.int32, (B, m), "Yhat"))
    if isinstance(W, PackedW):
        if path == "valu":
            raise ValueError("packed weights use the matrix-core kernels")
        _lib.check("mvk_server_eval_packed", L.mvk_server_eval_packed(W.data.data_ptr(), *tail, _stream(stream)))
        return out
    args = (_dev(W, torch.int8, (m, n), "W"),) + tail
    if path == "auto":
        _lib.check("mvk_server_eval", L.mvk_server_eval(*args, _stream(stream)))
    else:
        _lib.check("mvk_server_eval_path", L.mvk_server_eval_path(*args, PATHS[path], _stream(stream)))
    return out


def keygen(key: Key, W: torch.Tensor, stream=None) -> Key:
    """Preprocess: fills key.PT = (W Gx)^T and key.Q = Gy^T W."""
    _dev(W, torch.int8, (key.m, key.n), "W")
    ks = key.struct()
    _lib.check("mvk_keygen", _lib.load(key.p).mvk_keygen(ctypes.byref(ks), W.data_ptr(), _stream(stream)))
    return key


def encode(key: Key, X: torch.Tensor, ex_idx: torch.Tensor, ex_val: torch.Tensor,
           out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Encrypt: Xhat_b = X_b + Gx e_b.  X: B x n; ex_idx/ex_val: B x t_x."""
    B = X.shape[0]
    if out is None:
        out = torch.empty_like(X)
    ks = key.struct()
    ex = _sparse(ex_idx, ex_val, "ex")
    _lib.check("mvk_encode", _lib.load(key.p).mvk_encode(
        ctypes.byref(ks), _dev(X, torch.int32, (B, key.n), "X"), B, ctypes.byref(ex),
        _dev(out, torch.int32, (B, key.n), "Xhat"), _stream(stream)))
    return out


def verify_prepare(key: Key, ey_idx: torch.Tensor, ey_val: torch.Tensor, R: torch.Tensor | None = None,
                   stream=None) -> torch.Tensor:
    """Challenge syndromes R[q] = Gy e_q (ell x m) for decode_verify(..., R=R)."""
    ell = ey_idx.shape[0]
    if R is None:
        R = torch.empty((ell, key.m), dtype=torch.int32, device=ey_idx.device)
    ks = key.struct()
    ey = _sparse(ey_idx, ey_val, "ey")
    _lib.check("mvk_verify_prepare", _lib.load(key.p).mvk_verify_prepare(
        ctypes.byref(ks), ctypes.byref(ey), _dev(R, torch.int32, (ell, key.m), "R"), _stream(stream)))
    return R


def decode_verify(key: Key, Xhat: torch.Tensor, Yhat: torch.Tensor, ex_idx: torch.Tensor, ex_val: torch.Tensor,
                  ey_idx: torch.Tensor, ey_val: torch.Tensor, Y: torch.Tensor | None = None,
                  vL: torch.Tensor | None = None, vR: torch.Tensor | None = None,
                  accept: torch.Tensor | None = None, stream=None, R: torch.Tensor | None = None):
    """Verify + Decrypt.  Returns (Y, accept, vL, vR); accept is int32 0/1 per column.

    R: challenge syndromes from verify_prepare for the same ey (optional; when
    absent they are computed inside the call)."""
    B = Xhat.shape[0]
    ell = ey_idx.shape[0]
    dev = Xhat.device
    if Y is None:
        Y = torch.empty((B, key.m), dtype=torch.int32, device=dev)
    if accept is None:
        accept = torch.empty((B,), dtype=torch.int32, device=dev)
    ks = key.struct()
    ex = _sparse(ex_idx, ex_val, "ex")
    ey = _sparse(ey_idx, ey_val, "ey")
    vLp = _dev(vL, torch.int32, (ell, B), "vL") if vL is not None else None
    vRp = _dev(vR, torch.int32, (ell, B), "vR") if vR is not None else None
    common = (_dev(Xhat, torch.int32, (B, key.n), "Xhat"), _dev(Yhat, torch.int32, (B, key.m), "Yhat"),
              B, ctypes.byref(ex), ctypes.byref(ey))
    outs = (_dev(Y, torch.int32, (B, key.m), "Y"), vLp, vRp, _dev(accept, torch.int32, (B,), "accept"),
            _stream(stream))
    if R is None:
        _lib.check("mvk_decode_verify", _lib.load(key.p).mvk_decode_verify(ctypes.byref(ks), *common, *outs))
    else:
        _lib.check("mvk_decode_verify_prepared", _lib.load(key.p).mvk_decode_verify_prepared(
            ctypes.byref(ks), *common, _dev(R, torch.int32, (ell, key.m), "R"), *outs))
    return Y, accept, vL, vR


class Prepared:
    """Client preparation for one query batch (secret to the client): input and
    output masks of B noise vectors and the vectors of ell challenges."""

    def __init__(self, key: Key, B: int, ell: int, device="cuda"):
        i32 = dict(dtype=torch.int32, device=device)
        self.B, self.ell = B, ell
        self.Mx = torch.empty((B, key.n), **i32)
        self.My = torch.empty((B, key.m), **i32)
        self.R = torch.empty((ell, key.m), **i32)
        self.U = torch.empty((ell, key.n), **i32)


def client_prepare(key: Key, ex_idx: torch.Tensor, ex_val: torch.Tensor, ey_idx: torch.Tensor,
                   ey_val: torch.Tensor, out: Prepared | None = None, done_flag: torch.Tensor | None = None,
                   done_value: int = 1, stream=None) -> Prepared:
    """Masks Mx = Gx e_b, My = P e_b (per noise vector) and R = Gy e_q,
    U = e_q^T Q (per challenge): the query- and response-independent work.
    done_flag: device word set to done_value once every output is visible."""
    B, ell = ex_idx.shape[0], ey_idx.shape[0]
    if out is None:
        out = Prepared(key, B, ell, device=ex_idx.device)
    if (out.B, out.ell) != (B, ell):
        raise ValueError("Prepared buffers do not match the noise / challenge counts")
    ks = key.struct()
    ex = _sparse(ex_idx, ex_val, "ex")
    ey = _sparse(ey_idx, ey_val, "ey")
    _lib.check("mvk_client_prepare", _lib.load(key.p).mvk_client_prepare(
        ctypes.byref(ks), ctypes.byref(ex), ctypes.byref(ey),
        _dev(out.Mx, torch.int32, (B, key.n), "Mx"), _dev(out.My, torch.int32, (B, key.m), "My"),
        _dev(out.R, torch.int32, (ell, key.m), "R"), _dev(out.U, torch.int32, (ell, key.n), "U"),
        _dev(done_flag, torch.int32, (), "done_flag") if done_flag is not None else None, done_value,
        _stream(stream)))
    return out


def client_prepare_group(keys: list, ex_idx: torch.Tensor, ex_val: torch.Tensor, eys: list, outs: list | None = None,
                         done_flag: torch.Tensor | None = None, done_value: int = 1, stream=None) -> list:
    """client_prepare for several keys sharing the noise (one shape, one privacy
    code): the input mask once (in every returned Prepared), the output masks
    and challenge vectors per key.  eys: [(ey_idx, ey_val)] per key."""
    G = len(keys)
    B = ex_idx.shape[0]
    ell = eys[0][0].shape[0]
    if outs is None:
        outs = [Prepared(k, B, ell, device=ex_idx.device) for k in keys]
    if any((o.B, o.ell) != (B, ell) for o in outs):
        raise ValueError("Prepared buffers do not match the noise / challenge counts")
    structs = [k.struct() for k in keys]
    kp = (ctypes.POINTER(MvkKey) * G)(*[ctypes.pointer(ks) for ks in structs])
    ex = _sparse(ex_idx, ex_val, "ex")
    ey_structs = [_sparse(i, v, f"ey[{g}]") for g, (i, v) in enumerate(eys)]
    eyp = (ctypes.POINTER(MvkSparse) * G)(*[ctypes.pointer(e) for e in ey_structs])
    m, n = keys[0].m, keys[0].n
    # the shared input mask goes to the first Prepared; the others get a copy view of it
    arr = lambda ts, shape, name: (ctypes.c_void_p * G)(*[_dev(t, torch.int32, shape, f"{name}[{g}]")  # noqa: E731
                                                          for g, t in enumerate(ts)])
    _lib.check("mvk_client_prepare_group", _lib.load(keys[0].p).mvk_client_prepare_group(
        G, kp, ctypes.byref(ex), eyp, _dev(outs[0].Mx, torch.int32, (B, n), "Mx"),
        arr([o.My for o in outs], (B, m), "My"), arr([o.R for o in outs], (ell, m), "R"),
        arr([o.U for o in outs], (ell, n), "U"),
        _dev(done_flag, torch.int32, (), "done_flag") if done_flag is not None else None, done_value,
        _stream(stream)))
    for o in outs[1:]:
        o.Mx = outs[0].Mx
    return outs


def client_prepare_multi(keys: list, exs: list, eys: list, outs: list | None = None, done_flags: list | None = None,
                         done_value: int = 1, stream=None) -> list:
    """client_prepare for several keys and inputs in one call (one launch for
    the short syndromes and every row gather).  exs[g] = (ex_idx, ex_val) of
    key g's input, or None; eys[g] = (ey_idx, ey_val) or None.  Keys listed
    with the same noise tensors share their input: the input mask is computed
    once and every Prepared of that input holds the same Mx tensor.
    done_flags: None, or per key a device word (or None) set to done_value
    once every output of the call is visible."""
    G = len(keys)
    if not 1 <= G <= _lib.MVK_MAX_PREP or len(exs) != G or len(eys) != G:
        raise ValueError(f"1..{_lib.MVK_MAX_PREP} keys, with one noise and one challenge entry each")
    dev_ = next(t[0].device for t in list(exs) + list(eys) if t is not None)
    if outs is None:
        outs = [Prepared(k, exs[g][0].shape[0] if exs[g] is not None else 0,
                         eys[g][0].shape[0] if eys[g] is not None else 0, device=dev_) for g, k in enumerate(keys)]
    # one input mask per distinct noise: the first Prepared of that noise holds it
    owner = {}
    for g, e in enumerate(exs):
        if e is not None:
            k = (e[0].data_ptr(), e[1].data_ptr())
            if k in owner:
                outs[g].Mx = outs[owner[k]].Mx
            else:
                owner[k] = g
    structs = [k.struct() for k in keys]
    kp = (ctypes.POINTER(MvkKey) * G)(*[ctypes.pointer(ks) for ks in structs])
    ex_s = [_sparse(e[0], e[1], f"ex[{g}]") if e is not None else None for g, e in enumerate(exs)]
    ey_s = [_sparse(e[0], e[1], f"ey[{g}]") if e is not None else None for g, e in enumerate(eys)]
    exp = (ctypes.POINTER(MvkSparse) * G)(*[ctypes.pointer(e) if e is not None else None for e in ex_s])
    eyp = (ctypes.POINTER(MvkSparse) * G)(*[ctypes.pointer(e) if e is not None else None for e in ey_s])

    for g, o in enumerate(outs):
        if (exs[g] is not None and o.B != exs[g][0].shape[0]) or (eys[g] is not None and o.ell != eys[g][0].shape[0]):
            raise ValueError("Prepared buffers do not match the noise / challenge counts")

    def arr(name, pick):
        """Device pointers of one output per key; pick(g) -> (tensor, shape) or None."""
        ptrs = []
        for g in range(G):
            ts = pick(g)
            ptrs.append(_dev(ts[0], torch.int32, ts[1], f"{name}[{g}]") if ts is not None else None)
        return (ctypes.c_void_p * G)(*ptrs)

    ks_, os_ = keys, outs
    Mx = arr("Mx", lambda g: (os_[g].Mx, (os_[g].B, ks_[g].n)) if exs[g] is not None else None)
    My = arr("My", lambda g: (os_[g].My, (os_[g].B, ks_[g].m)) if exs[g] is not None else None)
    R = arr("R", lambda g: (os_[g].R, (os_[g].ell, ks_[g].m)) if eys[g] is not None else None)
    U = arr("U", lambda g: (os_[g].U, (os_[g].ell, ks_[g].n)) if eys[g] is not None else None)
    flags = None
    if done_flags is not None:
        flags = (ctypes.c_void_p * G)(*[_dev(f, torch.int32, (), f"done_flags[{g}]") if f is not None else None
                                        for g, f in enumerate(done_flags)])
    _lib.check("mvk_client_prepare_multi", _lib.load(keys[0].p).mvk_client_prepare_multi(
        G, kp, exp, eyp, Mx, My, R, U, flags, done_value, _stream(stream)))
    return outs


def encode_masked(key: Key, X: torch.Tensor, prep: Prepared, out: torch.Tensor | None = None,
                  ready_flag: torch.Tensor | None = None, ready_value: int = 1, timeout_us: int = 200000,
                  timed_out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Encrypt with a prepared mask: Xhat = X + Mx; with ready_flag, first wait
    for it to hold ready_value (see flag_wait)."""
    B = X.shape[0]
    if out is None:
        out = torch.empty_like(X)
    ks = key.struct()
    _lib.check("mvk_encode_masked", _lib.load(key.p).mvk_encode_masked(
        ctypes.byref(ks), _dev(X, torch.int32, (B, key.n), "X"), B,
        _dev(prep.Mx, torch.int32, (B, key.n), "Mx"), _dev(out, torch.int32, (B, key.n), "Xhat"),
        _dev(ready_flag, torch.int32, (), "ready_flag") if ready_flag is not None else None, ready_value,
        timeout_us, _dev(timed_out, torch.int32, (), "timed_out") if timed_out is not None else None,
        _stream(stream)))
    return out


def decode_verify_masked(key: Key, Xhat: torch.Tensor, Yhat: torch.Tensor, prep: Prepared,
                         Y: torch.Tensor | None = None, vL: torch.Tensor | None = None,
                         vR: torch.Tensor | None = None, accept: torch.Tensor | None = None, stream=None):
    """Verify + Decrypt with prepared masks and challenge vectors.  Returns (Y, accept, vL, vR)."""
    B, ell = Xhat.shape[0], prep.ell
    dev = Xhat.device
    if Y is None:
        Y = torch.empty((B, key.m), dtype=torch.int32, device=dev)
    if accept is None:
        accept = torch.empty((B,), dtype=torch.int32, device=dev)
    ks = key.struct()
    vLp = _dev(vL, torch.int32, (ell, B), "vL") if vL is not None else None
    vRp = _dev(vR, torch.int32, (ell, B), "vR") if vR is not None else None
    _lib.check("mvk_decode_verify_masked", _lib.load(key.p).mvk_decode_verify_masked(
        ctypes.byref(ks), _dev(Xhat, torch.int32, (B, key.n), "Xhat"), _dev(Yhat, torch.int32, (B, key.m), "Yhat"),
        B, _dev(prep.My, torch.int32, (B, key.m), "My"), ell, _dev(prep.R, torch.int32, (ell, key.m), "R"),
        _dev(prep.U, torch.int32, (ell, key.n), "U"), _dev(Y, torch.int32, (B, key.m), "Y"), vLp, vRp,
        _dev(accept, torch.int32, (B,), "accept"), _stream(stream)))
    return Y, accept, vL, vR


def decode_verify_encode_masked(key: Key, Xhat: torch.Tensor, Yhat: torch.Tensor, prep: Prepared,
                                X_next: torch.Tensor, prep_next: Prepared, Y: torch.Tensor | None = None,
                                vL: torch.Tensor | None = None, vR: torch.Tensor | None = None,
                                accept: torch.Tensor | None = None, out_next: torch.Tensor | None = None,
                                ready_flag: torch.Tensor | None = None, ready_value: int = 1,
                                timeout_us: int = 200000, timed_out: torch.Tensor | None = None, stream=None):
    """One client turn for independent queries: decode_verify_masked of this
    response and encode_masked of the next query (one launch where the
    decode/verify is small).  Returns (Y, accept, vL, vR, Xhat_next)."""
    B, ell = Xhat.shape[0], prep.ell
    Bn = X_next.shape[0]
    dev = Xhat.device
    if Y is None:
        Y = torch.empty((B, key.m), dtype=torch.int32, device=dev)
    if accept is None:
        accept = torch.empty((B,), dtype=torch.int32, device=dev)
    if out_next is None:
        out_next = torch.empty_like(X_next)
    ks = key.struct()
    vLp = _dev(vL, torch.int32, (ell, B), "vL") if vL is not None else None
    vRp = _dev(vR, torch.int32, (ell, B), "vR") if vR is not None else None
    _lib.check("mvk_decode_verify_encode_masked", _lib.load(key.p).mvk_decode_verify_encode_masked(
        ctypes.byref(ks), _dev(Xhat, torch.int32, (B, key.n), "Xhat"), _dev(Yhat, torch.int32, (B, key.m), "Yhat"),
        B, _dev(prep.My, torch.int32, (B, key.m), "My"), ell, _dev(prep.R, torch.int32, (ell, key.m), "R"),
        _dev(prep.U, torch.int32, (ell, key.n), "U"), _dev(Y, torch.int32, (B, key.m), "Y"), vLp, vRp,
        _dev(accept, torch.int32, (B,), "accept"), _dev(X_next, torch.int32, (Bn, key.n), "X_next"), Bn,
        _dev(prep_next.Mx, torch.int32, (Bn, key.n), "Mx_next"), _dev(out_next, torch.int32, (Bn, key.n), "Xhat_next"),
        _dev(ready_flag, torch.int32, (), "ready_flag") if ready_flag is not None else None, ready_value,
        timeout_us, _dev(timed_out, torch.int32, (), "timed_out") if timed_out is not None else None,
        _stream(stream)))
    return Y, accept, vL, vR, out_next


def decode_verify_masked_group(keys: list, Xhat: torch.Tensor, Yhats: list, preps: list, Ys: list | None = None,
                               vLs: list | None = None, vRs: list | None = None, accepts: list | None = None,
                               stream=None):
    """decode_verify_masked for several matrices sharing the queries Xhat (one
    launch where the problem allows).  Returns (Ys, accepts, vLs, vRs)."""
    G = len(keys)
    B = Xhat.shape[0]
    ell = preps[0].ell
    m, n = keys[0].m, keys[0].n
    dev = Xhat.device
    if Ys is None:
        Ys = [torch.empty((B, m), dtype=torch.int32, device=dev) for _ in range(G)]
    if accepts is None:
        accepts = [torch.empty((B,), dtype=torch.int32, device=dev) for _ in range(G)]
    structs = [k.struct() for k in keys]
    kp = (ctypes.POINTER(MvkKey) * G)(*[ctypes.pointer(ks) for ks in structs])

    def arr(ts, shape, name):
        return (ctypes.c_void_p * G)(*[_dev(t, torch.int32, shape, f"{name}[{g}]") for g, t in enumerate(ts)])

    if any(p.ell != ell for p in preps):
        raise ValueError("the prepared vectors of a group must have one repetition count")
    _lib.check("mvk_decode_verify_masked_group", _lib.load(keys[0].p).mvk_decode_verify_masked_group(
        G, kp, _dev(Xhat, torch.int32, (B, n), "Xhat"), B, arr(Yhats, (B, m), "Yhat"),
        arr([p.My for p in preps], (B, m), "My"), ell, arr([p.R for p in preps], (ell, m), "R"),
        arr([p.U for p in preps], (ell, n), "U"), arr(Ys, (B, m), "Y"),
        arr(vLs, (ell, B), "vL") if vLs is not None else None, arr(vRs, (ell, B), "vR") if vRs is not None else None,
        arr(accepts, (B,), "accept"), _stream(stream)))
    return Ys, accepts, vLs, vRs


class CUStream:
    """A stream restricted to the compute units [first_cu, first_cu + count)
    (mvk_stream_create_cu_range); .stream is the torch view of it.  The HIP
    stream is destroyed by close() (or when this object is collected), after
    the device has finished its work."""

    def __init__(self, first_cu: int, count: int):
        h = ctypes.c_void_p()
        _lib.check("mvk_stream_create_cu_range", _lib.load().mvk_stream_create_cu_range(first_cu, count,
                                                                                          ctypes.byref(h)))
        self._h = h.value
        self.first_cu, self.count = first_cu, count
        self.stream = torch.cuda.ExternalStream(self._h)

    def close(self) -> None:
        if self._h:
            torch.cuda.synchronize()
            _lib.check("mvk_stream_destroy", _lib.load().mvk_stream_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def device_cus() -> int:
    """Compute units of the current device."""
    return torch.cuda.get_device_properties(torch.cuda.current_device()).multi_processor_count


def flag_signal(flag: torch.Tensor, value: int = 1, stream=None) -> None:
    """Set the device word `flag` to value once the stream's earlier work is done."""
    _lib.check("mvk_flag_signal", _lib.load().mvk_flag_signal(
        _dev(flag, torch.int32, (), "flag"), value, _stream(stream)))


def flag_wait(flag: torch.Tensor, value: int = 1, timeout_us: int = 200000, timed_out: torch.Tensor | None = None,
              stream=None) -> None:
    """Make the stream wait until flag == value (then clear it); on time-out set timed_out."""
    _lib.check("mvk_flag_wait", _lib.load().mvk_flag_wait(
        _dev(flag, torch.int32, (), "flag"), value, timeout_us,
        _dev(timed_out, torch.int32, (), "timed_out") if timed_out is not None else None, _stream(stream)))


def verify(key: Key, X: torch.Tensor, Y: torch.Tensor, ey_idx: torch.Tensor, ey_val: torch.Tensor,
           vL: torch.Tensor | None = None, vR: torch.Tensor | None = None, accept: torch.Tensor | None = None,
           stream=None):
    """Verification only (vMVMD): check Y = W X for plaintext X (B x n) and Y (B x m).
    Returns (accept, vL, vR); accept is int32 0/1 per column."""
    B, ell = X.shape[0], ey_idx.shape[0]
    if accept is None:
        accept = torch.empty((B,), dtype=torch.int32, device=X.device)
    ks = key.struct()
    ey = _sparse(ey_idx, ey_val, "ey")
    _lib.check("mvk_verify", _lib.load(key.p).mvk_verify(
        ctypes.byref(ks), _dev(X, torch.int32, (B, key.n), "X"), _dev(Y, torch.int32, (B, key.m), "Y"), B,
        ctypes.byref(ey), _dev(vL, torch.int32, (ell, B), "vL") if vL is not None else None,
        _dev(vR, torch.int32, (ell, B), "vR") if vR is not None else None,
        _dev(accept, torch.int32, (B,), "accept"), _stream(stream)))
    return accept, vL, vR


def batch_preprocess(Qs: list, c2: Code, stream=None):
    """Batch verification, preprocessing: Qs = [Q_1, ..., Q_B] (N x n each, from
    keygen with one verification code); returns (QtT (N x Bn), Qaux (N x N'))."""
    B = len(Qs)
    N, n = Qs[0].shape
    ptrs = (ctypes.c_void_p * B)(*[_dev(Q, torch.int32, (N, n), f"Q[{b}]") for b, Q in enumerate(Qs)])
    dev = Qs[0].device
    QtT = torch.empty((N, B * n), dtype=torch.int32, device=dev)
    Qaux = torch.empty((N, c2.N), dtype=torch.int32, device=dev)
    cs = c2.struct()
    _lib.check("mvk_batch_preprocess", _lib.load(c2.p).mvk_batch_preprocess(
        B, ptrs, N, n, ctypes.byref(cs), QtT.data_ptr(), Qaux.data_ptr(), _stream(stream)))
    return QtT, Qaux


def batch_project(QtT: torch.Tensor, n: int, e_idx: torch.Tensor, e_val: torch.Tensor,
                  out: torch.Tensor | None = None, stream=None, p: int = P) -> torch.Tensor:
    """Batch verification, server step: Ut[q] = Qt e_q (ell x Bn)."""
    N, Bn = QtT.shape
    B = Bn // n
    ell = e_idx.shape[0]
    if out is None:
        out = torch.empty((ell, Bn), dtype=torch.int32, device=QtT.device)
    e = _sparse(e_idx, e_val, "e")
    _lib.check("mvk_batch_project", _lib.load(p).mvk_batch_project(
        _dev(QtT, torch.int32, (N, Bn), "QtT"), N, n, B, ctypes.byref(e),
        _dev(out, torch.int32, (ell, Bn), "Ut"), _stream(stream)))
    return out


def batch_verify(cy: Code, c2: Code, Qaux: torch.Tensor, X: torch.Tensor, Y: torch.Tensor, e_idx: torch.Tensor,
                 e_val: torch.Tensor, Ut: torch.Tensor, e2_idx: torch.Tensor, e2_val: torch.Tensor,
                 accept: torch.Tensor | None = None, vL=None, vR=None, sL=None, sR=None, stream=None):
    """Batch verification, client checks.  Returns (accept, vL, vR, sL, sR)."""
    B, n = X.shape
    m = Y.shape[1]
    ell, ell2 = e_idx.shape[0], e2_idx.shape[0]
    if accept is None:
        accept = torch.empty((B,), dtype=torch.int32, device=X.device)
    if cy.p != c2.p:
        raise ValueError("the two codes must be over one field")
    c1s, c2s = cy.struct(), c2.struct()
    e, e2 = _sparse(e_idx, e_val, "e"), _sparse(e2_idx, e2_val, "e2")
    opt = lambda t, shape, name: _dev(t, torch.int32, shape, name) if t is not None else None  # noqa: E731
    _lib.check("mvk_batch_verify", _lib.load(cy.p).mvk_batch_verify(
        ctypes.byref(c1s), ctypes.byref(c2s), _dev(Qaux, torch.int32, (cy.N, c2.N), "Qaux"), m, n, B,
        _dev(X, torch.int32, (B, n), "X"), _dev(Y, torch.int32, (B, m), "Y"), ctypes.byref(e),
        _dev(Ut, torch.int32, (ell, B * n), "Ut"), ctypes.byref(e2), opt(vL, (ell, B), "vL"), opt(vR, (ell, B), "vR"),
        opt(sL, (ell, ell2), "sL"), opt(sR, (ell, ell2), "sR"), _dev(accept, torch.int32, (B,), "accept"),
        _stream(stream)))
    return accept, vL, vR, sL, sR


def raa_encode(code: Code, w: torch.Tensor, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """G^T w for each row of w (count x k) -> count x N."""
    w2 = w if w.dim() == 2 else w.reshape(1, -1)
    count = w2.shape[0]
    if out is None:
        out = torch.empty((count, code.N), dtype=torch.int32, device=w.device)
    cs = code.struct()
    _lib.check("mvk_raa_encode", _lib.load(code.p).mvk_raa_encode(
        ctypes.byref(cs), _dev(w2, torch.int32, (count, code.k), "w"), count,
        _dev(out, torch.int32, (count, code.N), "out"), _stream(stream)))
    return out


def raa_syndrome(code: Code, v: torch.Tensor, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """G v for each row of v (count x N) -> count x k."""
    v2 = v if v.dim() == 2 else v.reshape(1, -1)
    count = v2.shape[0]
    if out is None:
        out = torch.empty((count, code.k), dtype=torch.int32, device=v.device)
    cs = code.struct()
    _lib.check("mvk_raa_syndrome", _lib.load(code.p).mvk_raa_syndrome(
        ctypes.byref(cs), _dev(v2, torch.int32, (count, code.N), "v"), count,
        _dev(out, torch.int32, (count, code.k), "out"), _stream(stream)))
    return out


def stream_read(data: torch.Tensor, sink: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Streaming read of a contiguous device tensor (its bytes, a multiple of 16,
    16-byte aligned): the HBM read floor for that size.  Returns the sink
    (MVK_STREAM_READ_BLOCKS int32 words whose XOR is the XOR of the buffer's
    32-bit words)."""
    if not data.is_cuda or not data.is_contiguous():
        raise ValueError("data must be a contiguous CUDA tensor")
    if sink is None:
        sink = torch.empty((_lib.MVK_STREAM_READ_BLOCKS,), dtype=torch.int32, device=data.device)
    nbytes = data.numel() * data.element_size()
    _lib.check("mvk_stream_read", _lib.load().mvk_stream_read(
        data.data_ptr(), nbytes, _dev(sink, torch.int32, (_lib.MVK_STREAM_READ_BLOCKS,), "sink"), _stream(stream)))
    return sink


# ---------------------------------------------------------------------------
# Seeded calls: the library draws the codes, the noise and the challenges
# ---------------------------------------------------------------------------
TAG_CODE_X = _lib.MVK_TAG_CODE_X
TAG_CODE_Y = _lib.MVK_TAG_CODE_Y
TAG_NOISE = _lib.MVK_TAG_NOISE
TAG_CHALLENGE = _lib.MVK_TAG_CHALLENGE
SEED_FRESH = _lib.MVK_SEED_FRESH


class _DeviceArray:
    """A library-owned int32 device array, seen by torch through the CUDA
    array interface (no copy; the owner keeps the memory alive)."""

    def __init__(self, ptr: int, shape: tuple):
        self.__cuda_array_interface__ = {"shape": tuple(int(d) for d in shape), "typestr": "<i4",
                                         "data": (int(ptr), False), "version": 2, "strides": None}


def _view(ptr: int, shape: tuple, device) -> torch.Tensor:
    if int(np_prod(shape)) == 0:
        return torch.empty(shape, dtype=torch.int32, device=device)
    return torch.as_tensor(_DeviceArray(ptr, shape), device=device)


def np_prod(shape) -> int:
    out = 1
    for d in shape:
        out *= int(d)
    return out


class SeededPP:
    """pp of Preprocess with library-drawn codes (mvk_keygen_seeded).  ``key`` is
    a Key whose tensors view the library's memory; every call that takes a Key
    accepts it.  The memory is freed when this object is collected."""

    def __init__(self, handle: int, p: int, device):
        self._handle, self._p = handle, p
        ks = _lib.load(p).mvk_pp_key(handle).contents
        cx, cy, m, n = ks.cx, ks.cy, ks.m, ks.n

        def code(c):
            N = c.k * c.r
            return Code(c.k, c.r, _view(c.pi1, (N,), device), _view(c.pi2, (N,), device), _view(c.v1, (N,), device),
                        _view(c.v2, (N,), device), p)

        self.key = Key(m, n, code(cx), code(cy), _view(ks.PT, (cx.k * cx.r, m), device),
                       _view(ks.Q, (cy.k * cy.r, n), device))
        self.key._owner = self

    def __del__(self):
        h, self._handle = getattr(self, "_handle", None), None
        if h:
            _lib.load(self._p).mvk_pp_free(h)


class SeededState:
    """st of Encrypt with library-drawn noise (mvk_encode_seeded): ``idx``,
    ``val`` (B x t_x) view the library's device arrays."""

    def __init__(self, handle: int, p: int, device):
        self._handle, self._p = handle, p
        sp = _lib.load(p).mvk_st_noise(handle).contents
        self.B, self.t = sp.count, sp.t
        self.idx = _view(sp.idx or 0, (sp.count, sp.t), device)
        self.val = _view(sp.val or 0, (sp.count, sp.t), device)

    def __del__(self):
        h, self._handle = getattr(self, "_handle", None), None
        if h:
            _lib.load(self._p).mvk_st_free(h)


def keygen_seeded(W: torch.Tensor, r_x: int, r_y: int, code_seed: int, p: int = P, stream=None) -> SeededPP:
    """Preprocess with codes drawn from code_seed (SEED_FRESH: from the OS)."""
    m, n = W.shape
    out = ctypes.c_void_p()
    _lib.check("mvk_keygen_seeded", _lib.load(p).mvk_keygen_seeded(
        m, n, r_x, r_y, code_seed & 0xFFFFFFFFFFFFFFFF, _dev(W, torch.int8, (m, n), "W"), _stream(stream),
        ctypes.byref(out)))
    return SeededPP(out.value, p, W.device)


def encode_seeded(key: Key, X: torch.Tensor, t_x: int, noise_seed: int, out: torch.Tensor | None = None,
                  stream=None):
    """Encrypt with noise drawn from noise_seed: returns (Xhat, SeededState)."""
    B = X.shape[0]
    if out is None:
        out = torch.empty_like(X)
    ks = key.struct()
    h = ctypes.c_void_p()
    _lib.check("mvk_encode_seeded", _lib.load(key.p).mvk_encode_seeded(
        ctypes.byref(ks), _dev(X, torch.int32, (B, key.n), "X"), B, t_x, noise_seed & 0xFFFFFFFFFFFFFFFF,
        _dev(out, torch.int32, (B, key.n), "Xhat"), ctypes.byref(h), _stream(stream)))
    return out, SeededState(h.value, key.p, X.device)


def decode_verify_seeded(key: Key, st: SeededState, Xhat: torch.Tensor, Yhat: torch.Tensor, t_y: int, ell: int,
                         chal_seed: int, Y: torch.Tensor | None = None, vL: torch.Tensor | None = None,
                         vR: torch.Tensor | None = None, accept: torch.Tensor | None = None, stream=None):
    """Verify + Decrypt with ell challenges drawn from chal_seed.  Returns (Y, accept, vL, vR)."""
    B = st.B
    dev = Xhat.device
    if Y is None:
        Y = torch.empty((B, key.m), dtype=torch.int32, device=dev)
    if accept is None:
        accept = torch.empty((B,), dtype=torch.int32, device=dev)
    ks = key.struct()
    _lib.check("mvk_decode_verify_seeded", _lib.load(key.p).mvk_decode_verify_seeded(
        ctypes.byref(ks), st._handle, _dev(Xhat, torch.int32, (B, key.n), "Xhat"),
        _dev(Yhat, torch.int32, (B, key.m), "Yhat"), t_y, ell, chal_seed & 0xFFFFFFFFFFFFFFFF,
        _dev(Y, torch.int32, (B, key.m), "Y"), _dev(vL, torch.int32, (ell, B), "vL") if vL is not None else None,
        _dev(vR, torch.int32, (ell, B), "vR") if vR is not None else None, _dev(accept, torch.int32, (B,), "accept"),
        _stream(stream)))
    return Y, accept, vL, vR


def sample_code(k: int, r: int, seed: int, tag: int, p: int = P) -> dict:
    """The library's host draw of a code (k, r): dict(k, r, N, pi1, pi2, v1, v2) of uint32 numpy arrays."""
    import numpy as np
    N = k * r
    arrs = [np.empty(N, dtype=np.uint32) for _ in range(4)]
    ptr = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))  # noqa: E731
    _lib.check("mvk_sample_code", _lib.load(p).mvk_sample_code(k, r, seed & 0xFFFFFFFFFFFFFFFF, tag,
                                                               *[ptr(a) for a in arrs]))
    return dict(k=k, r=r, N=N, pi1=arrs[0], pi2=arrs[1], v1=arrs[2], v2=arrs[3])


def sample_sparse(count: int, N: int, t: int, seed: int, tag: int, p: int = P):
    """The library's host draw of ``count`` vectors of E_t^N: (idx, val), uint32 numpy count x t."""
    import numpy as np
    idx = np.empty((count, t), dtype=np.uint32)
    val = np.empty((count, t), dtype=np.uint32)
    ptr = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))  # noqa: E731
    _lib.check("mvk_sample_sparse", _lib.load(p).mvk_sample_sparse(count, N, t, seed & 0xFFFFFFFFFFFFFFFF, tag,
                                                                   ptr(idx), ptr(val)))
    return idx, val
