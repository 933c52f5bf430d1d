"""CPU oracle for the pvMVMD hot path (Maverick, arxiv 2609.10264).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the bench's CPU
baseline leg are the only callers.  The product library shares no code with
this package and never imports it.

The arithmetic lives in ``mvk_oracle.c`` (plain C, '%' on uint64); this module
only builds it with gcc, loads it with ctypes and marshals numpy arrays.  The C
file is built once per field (``-DORC_P``): p = 2^31 - 1 (``P``, the default
of every function) and the BabyBear prime 15 * 2^27 + 1 (``P_BABYBEAR``, the
field of Sec. 7.1); every function takes the field as its ``p`` argument.  The
parameter helpers below restate the paper's formulas (Eq. (1) and Theorem 6.1).

Parity status per function:
  encT, syn          pinned: dense factor-matrix product of App. B, closed forms,
                     linearity, transposition identity
  server_eval        pinned: Python big-integer brute force, closed forms
  keygen             pinned: P = W Gx and Q = Gy^T W against dense G
  encode, decode     pinned: completeness (decode(server(encode(x))) = W x)
  verify             pinned: completeness, tamper rejection, exact acceptance
                     probability of Lemma 5.1 for t = 1
  noise_weight, verify_params
                     pinned: the values printed in Sec. 7.1
  batch_aux, batch_project, batch_verify
                     pinned: dense Qt^T G' and the secondary identity with
                     dense matrices, completeness, rejection of a wrong claim,
                     of a wrong projection and of a consistent forgery
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
import threading

import numpy as np

P = 2**31 - 1
P_BABYBEAR = 15 * 2**27 + 1
_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mvk_oracle.c")
_LIBS = {P: os.path.join(_HERE, "libmvk_oracle.so"), P_BABYBEAR: os.path.join(_HERE, "libmvk_oracle_bb.so")}
_lock = threading.Lock()
_lib = {}


def build(force: bool = False) -> list:
    """Compile the oracle with gcc, once per field (no GPU code involved)."""
    for p, path in _LIBS.items():
        if force or not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_SRC):
            tmp = path + ".tmp%d" % os.getpid()
            subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", f"-DORC_P={p}ULL", "-o", tmp,
                                   _SRC])
            os.replace(tmp, path)
    return list(_LIBS.values())


def configure(L) -> None:
    """Argument and result types of every oracle entry point on a loaded library."""
    u32p = ctypes.POINTER(ctypes.c_uint32)
    i8p = ctypes.POINTER(ctypes.c_int8)
    u8p = ctypes.POINTER(ctypes.c_uint8)
    u32 = ctypes.c_uint32
    L.orc_encT.argtypes = [u32, u32, u32p, u32p, u32p, u32p, u32p, u32p]
    L.orc_syn.argtypes = [u32, u32, u32p, u32p, u32p, u32p, u32p, u32p]
    L.orc_server_eval.argtypes = [i8p, u32, u32, u32p, u32, u32p]
    L.orc_server_eval_rows.argtypes = [i8p, u32, u32, u32p, u32, u32p, u32, u32]
    L.orc_keygen.argtypes = [i8p, u32, u32, u32, u32p, u32p, u32p, u32p,
                             u32, u32p, u32p, u32p, u32p, u32p, u32p]
    L.orc_encode.argtypes = [u32, u32, u32p, u32p, u32p, u32p, u32p, u32, u32p, u32p, u32, u32p]
    L.orc_decode.argtypes = [u32p, u32, u32p, u32, u32p, u32p, u32, u32p]
    L.orc_batch_aux.argtypes = [u32, u32, u32, u32p, u32, u32p, u32p, u32p, u32p, u32p]
    L.orc_batch_project.argtypes = [u32, u32, u32, u32p, u32p, u32p, u32, u32, u32p]
    L.orc_batch_verify.argtypes = [u32, u32, u32, u32, u32p, u32p, u32p, u32p, u32, u32p, u32p, u32p, u32p,
                                   u32p, u32p, u32p, u32p, u32p, u32, u32, u32p, u32p, u32p, u32, u32,
                                   u32p, u32p, u32p, u32p]
    L.orc_verify.argtypes = [u32, u32, u32, u32p, u32p, u32p, u32p, u32p, u32p, u32p, u32,
                             u32p, u32p, u32, u32, u32p, u32p, u8p]
    L.orc_prime.restype = u32
    L.orc_ops_reset.argtypes = []
    L.orc_ops_count.argtypes = []
    L.orc_ops_count.restype = ctypes.c_uint64


def lib(p: int = P):
    with _lock:
        if p not in _lib:
            if p not in _LIBS:
                raise ValueError(f"no oracle build over p = {p}")
            build()
            L = ctypes.CDLL(_LIBS[p])
            configure(L)
            assert L.orc_prime() == p
            _lib[p] = L
    return _lib[p]


def _u32(a) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.uint32)
    return a


def _p(a, ct=ctypes.c_uint32):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ct))


def _code_args(code):
    arrs = [_u32(code[k]) for k in ("pi1", "pi2", "v1", "v2")]
    return arrs


# ---------------------------------------------------------------------------
# RAA code maps (App. B)
# ---------------------------------------------------------------------------
def encT(code: dict, w, p: int = P) -> np.ndarray:
    """G^T w for w in F^k (App. B, linear-time encoding)."""
    k, r = code["k"], code["r"]
    w = _u32(w)
    assert w.shape == (k,)
    c = _code_args(code)
    out = np.empty(k * r, dtype=np.uint32)
    lib(p).orc_encT(k, r, *[_p(a) for a in c], _p(w), _p(out))
    return out


def field_ops(fn, p: int = P) -> int:
    """Field operations the oracle performs while fn() runs (fn calls the oracle
    over the same field)."""
    L = lib(p)
    L.orc_ops_reset()
    fn()
    return int(L.orc_ops_count())


def syn(code: dict, v, p: int = P) -> np.ndarray:
    """G v for v in F^N (App. B, syndrome by the transposition principle)."""
    k, r = code["k"], code["r"]
    v = _u32(v)
    assert v.shape == (k * r,)
    c = _code_args(code)
    out = np.empty(k, dtype=np.uint32)
    lib(p).orc_syn(k, r, *[_p(a) for a in c], _p(v), _p(out))
    return out


# ---------------------------------------------------------------------------
# Protocol pvMVMD
# ---------------------------------------------------------------------------
def server_eval(W, Xhat, rows=None, p: int = P) -> np.ndarray:
    """Yhat = W Xhat mod p; W int8 m x n, Xhat uint32 B x n -> uint32 B x m.

    ``rows`` = (row0, row1) restricts the computation to a row range (other
    entries of the result are left zero).
    """
    W = np.ascontiguousarray(W, dtype=np.int8)
    Xhat = _u32(np.atleast_2d(Xhat))
    m, n = W.shape
    B = Xhat.shape[0]
    assert Xhat.shape == (B, n)
    Y = np.zeros((B, m), dtype=np.uint32)
    if rows is None:
        lib(p).orc_server_eval(_p(W, ctypes.c_int8), m, n, _p(Xhat), B, _p(Y))
    else:
        lib(p).orc_server_eval_rows(_p(W, ctypes.c_int8), m, n, _p(Xhat), B, _p(Y), int(rows[0]), int(rows[1]))
    return Y


def keygen(W, cx: dict, cy: dict, want_P: bool = True, want_Q: bool = True, p: int = P):
    """Preprocess: returns (PT, Q) with PT = (W Gx)^T (Nx x m), Q = Gy^T W (Ny x n)."""
    W = np.ascontiguousarray(W, dtype=np.int8)
    m, n = W.shape
    assert cx["k"] == n and cy["k"] == m
    PT = np.empty((cx["N"], m), dtype=np.uint32) if want_P else None
    Q = np.empty((cy["N"], n), dtype=np.uint32) if want_Q else None
    ax = _code_args(cx)
    ay = _code_args(cy)
    lib(p).orc_keygen(_p(W, ctypes.c_int8), m, n, cx["r"], *[_p(a) for a in ax],
                     cy["r"], *[_p(a) for a in ay], _p(PT), _p(Q))
    return PT, Q


def encode(cx: dict, X, ex_idx, ex_val, p: int = P) -> np.ndarray:
    """Encrypt: Xhat = X + Gx e_x (per column); X uint32 B x n."""
    X = _u32(np.atleast_2d(X))
    B, n = X.shape
    assert cx["k"] == n
    ex_idx = _u32(ex_idx)
    ex_val = _u32(ex_val)
    tx = ex_idx.shape[1]
    assert ex_idx.shape == (B, tx) and ex_val.shape == (B, tx)
    Xhat = np.empty_like(X)
    a = _code_args(cx)
    lib(p).orc_encode(n, cx["r"], *[_p(x) for x in a], _p(X), B, _p(ex_idx), _p(ex_val), tx, _p(Xhat))
    return Xhat


def decode(PT, Yhat, ex_idx, ex_val, p: int = P) -> np.ndarray:
    """Decrypt: Y = Yhat - P e_x."""
    PT = _u32(PT)
    Yhat = _u32(np.atleast_2d(Yhat))
    B, m = Yhat.shape
    assert PT.shape[1] == m
    ex_idx = _u32(ex_idx)
    ex_val = _u32(ex_val)
    tx = ex_idx.shape[1]
    assert int(ex_idx.max(initial=0)) < PT.shape[0]
    Y = np.empty_like(Yhat)
    lib(p).orc_decode(_p(PT), m, _p(Yhat), B, _p(ex_idx), _p(ex_val), tx, _p(Y))
    return Y


def verify(cy: dict, Q, Xhat, Yhat, ey_idx, ey_val, p: int = P):
    """Verify: returns (accept[B] bool, vL[ell, B], vR[ell, B])."""
    Q = _u32(Q)
    Xhat = _u32(np.atleast_2d(Xhat))
    Yhat = _u32(np.atleast_2d(Yhat))
    B, n = Xhat.shape
    m = Yhat.shape[1]
    assert cy["k"] == m and Q.shape == (cy["N"], n) and Yhat.shape[0] == B
    ey_idx = _u32(np.atleast_2d(ey_idx))
    ey_val = _u32(np.atleast_2d(ey_val))
    ell, ty = ey_idx.shape
    vL = np.empty((ell, B), dtype=np.uint32)
    vR = np.empty((ell, B), dtype=np.uint32)
    acc = np.empty(B, dtype=np.uint8)
    a = _code_args(cy)
    lib(p).orc_verify(m, n, cy["r"], *[_p(x) for x in a], _p(Q), _p(Xhat), _p(Yhat), B,
                     _p(ey_idx), _p(ey_val), ty, ell, _p(vL), _p(vR), _p(acc, ctypes.c_uint8))
    return acc.astype(bool), vL, vR


# ---------------------------------------------------------------------------
# Protocol Batch-vMVMD (Sec. 5.4)
# ---------------------------------------------------------------------------
def batch_aux(Qs, c2: dict, p: int = P) -> np.ndarray:
    """Preprocess: Qaux = Qt^T G' (N x N') for Qs = [Q_1, ..., Q_B] (B x N x n)."""
    Qs = _u32(Qs)
    B, N, n = Qs.shape
    assert c2["k"] == B * n
    a = _code_args(c2)
    out = np.empty((N, c2["N"]), dtype=np.uint32)
    lib(p).orc_batch_aux(B, N, n, _p(Qs), c2["r"], *[_p(x) for x in a], _p(out))
    return out


def batch_project(Qs, e_idx, e_val, p: int = P) -> np.ndarray:
    """Server step: u~(q) = Qt e(q) (ell x Bn)."""
    Qs = _u32(Qs)
    B, N, n = Qs.shape
    e_idx = _u32(np.atleast_2d(e_idx))
    e_val = _u32(np.atleast_2d(e_val))
    ell, t = e_idx.shape
    assert int(e_idx.max(initial=0)) < N
    out = np.empty((ell, B * n), dtype=np.uint32)
    lib(p).orc_batch_project(B, N, n, _p(Qs), _p(e_idx), _p(e_val), t, ell, _p(out))
    return out


def batch_verify(cy: dict, c2: dict, Qaux, X, Y, e_idx, e_val, ut, e2_idx, e2_val, p: int = P):
    """Client checks.  Returns (accept[B] bool, batch_ok bool, vL, vR (ell x B),
    sL, sR (ell x ell2)); claim b is accepted iff every secondary check of the
    batch and every original check of b passes."""
    X = _u32(np.atleast_2d(X))
    Y = _u32(np.atleast_2d(Y))
    B, n = X.shape
    m = Y.shape[1]
    assert cy["k"] == m and c2["k"] == B * n and Y.shape[0] == B
    Qaux = _u32(Qaux)
    assert Qaux.shape == (cy["N"], c2["N"])
    e_idx, e_val = _u32(np.atleast_2d(e_idx)), _u32(np.atleast_2d(e_val))
    e2_idx, e2_val = _u32(np.atleast_2d(e2_idx)), _u32(np.atleast_2d(e2_val))
    ell, t = e_idx.shape
    ell2, t2 = e2_idx.shape
    ut = _u32(ut)
    assert ut.shape == (ell, B * n)
    vL = np.empty((ell, B), dtype=np.uint32)
    vR = np.empty((ell, B), dtype=np.uint32)
    sL = np.empty((ell, ell2), dtype=np.uint32)
    sR = np.empty((ell, ell2), dtype=np.uint32)
    a, a2 = _code_args(cy), _code_args(c2)
    lib(p).orc_batch_verify(m, n, B, cy["r"], *[_p(x) for x in a], c2["r"], *[_p(x) for x in a2], _p(Qaux),
                           _p(X), _p(Y), _p(e_idx), _p(e_val), t, ell, _p(ut), _p(e2_idx), _p(e2_val), t2, ell2,
                           _p(vL), _p(vR), _p(sL), _p(sR))
    batch_ok = bool((sL == sR).all())
    accept = (vL == vR).all(axis=0) & batch_ok
    return accept, batch_ok, vL, vR, sL, sR


# ---------------------------------------------------------------------------
# Parameter formulas
# ---------------------------------------------------------------------------
def noise_weight(lam: int, N: int, delta: float) -> int:
    """Eq. (1): smallest integer t with t >= ln2 * (lambda - log2 N) / delta."""
    return int(math.ceil(math.log(2) * (lam - math.log2(N)) / delta))


def verify_params(field_size: int, kappa: int, delta: float) -> tuple[int, int]:
    """(t, ell) for the sparse coded check.

    ell is Theorem 5.2's repetition count ceil(kappa / (log2(|F|-1) - 1)).
    t is the sparsity that the theorem's soundness case applies with: when
    1/(|F|-1) > 2^-(kappa+1) (every field of at most 41 bits) the proof only
    needs (1-delta)^t <= 1/(|F|-1), i.e. t = ceil(log2(|F|-1) / -log2(1-delta));
    otherwise t = ceil((kappa+1) / -log2(1-delta)) with ell = 1.
    """
    lf = math.log2(field_size - 1)
    d = -math.log2(1.0 - delta)
    if 1.0 / (field_size - 1) > 2.0 ** (-(kappa + 1)):
        return int(math.ceil(lf / d)), int(math.ceil(kappa / (lf - 1)))
    return int(math.ceil((kappa + 1) / d)), 1
