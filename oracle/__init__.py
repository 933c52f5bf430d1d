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
  sample_code, sample_sparse
                     the seeded sampling specification (the paper leaves the
                     generator open): pinned by the statistics its draws must
                     have (uniform permutations and F_p^* values, E_t^N
                     support), by SplitMix64's published reference outputs,
                     and by Lemma 5.1's exact acceptance probability with
                     challenges drawn this way
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
from concurrent.futures import ThreadPoolExecutor

import numpy as np

P = 2**31 - 1
P_BABYBEAR = 15 * 2**27 + 1
_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mvk_oracle.c")
# (prime, counting build) -> shared object.  The counting build keeps a global
# count of field operations (single-threaded use: the cost pins of App. B).
_LIBS = {(P, False): os.path.join(_HERE, "libmvk_oracle.so"),
         (P_BABYBEAR, False): os.path.join(_HERE, "libmvk_oracle_bb.so"),
         (P, True): os.path.join(_HERE, "libmvk_oracle_count.so"),
         (P_BABYBEAR, True): os.path.join(_HERE, "libmvk_oracle_bb_count.so")}
_lock = threading.Lock()
_count_lock = threading.Lock()  # one counted call at a time
_lib = {}
_lib_count = {}


def build(force: bool = False) -> list:
    """Compile the oracle with gcc, once per field and counting mode (no GPU
    code involved)."""
    for (p, count), path in _LIBS.items():
        if force or not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_SRC):
            tmp = path + ".tmp%d" % os.getpid()
            flags = ["-DORC_COUNT_OPS"] if count else []
            subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", f"-DORC_P={p}ULL", *flags, "-o",
                                   tmp, _SRC])
            os.replace(tmp, path)
    return list(_LIBS.values())


def threads() -> int:
    """Host threads the oracle's row-block helpers use: every core this
    process may run on, capped by OMP_NUM_THREADS when that is set."""
    try:
        n = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        n = os.cpu_count() or 1
    cap = os.environ.get("OMP_NUM_THREADS", "")
    if cap.isdigit() and int(cap) > 0:
        n = min(n, int(cap))
    return max(1, n)


def _blocks(total: int, nthreads: int, min_block: int = 1) -> list:
    """Split [0, total) into at most 4 * nthreads contiguous ranges."""
    if total <= 0:
        return []
    parts = max(1, min(4 * nthreads, total // max(1, min_block)))
    step = -(-total // parts)
    return [(a, min(total, a + step)) for a in range(0, total, step)]


def _run_blocks(fn, ranges, nthreads: int) -> None:
    """fn(a, b) over every range; several at once (ctypes releases the GIL
    while the C code runs, and the ranges write disjoint outputs)."""
    if nthreads <= 1 or len(ranges) <= 1:
        for a, b in ranges:
            fn(a, b)
        return
    with ThreadPoolExecutor(max_workers=nthreads) as ex:
        list(ex.map(lambda r: fn(*r), ranges))


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
    L.orc_keygen_PT_rows.argtypes = [i8p, u32, u32, u32, u32p, u32p, u32p, u32p, u32p, u32, u32]
    L.orc_keygen_Q_cols.argtypes = [i8p, u32, u32, u32, u32p, u32p, u32p, u32p, u32p, u32, u32]
    u64 = ctypes.c_uint64
    L.orc_sample_code.argtypes = [u32, u32, u64, u64, u32p, u32p, u32p, u32p]
    L.orc_sample_sparse.argtypes = [u32, u32, u32, u64, u64, u32p, u32p]
    L.orc_sm64_draws.argtypes = [u64, u32, ctypes.POINTER(u64)]
    L.orc_counts_ops.restype = ctypes.c_int
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


def lib(p: int = P, count: bool = False):
    """The oracle built over F_p (count: the counting build)."""
    cache = _lib_count if count else _lib
    with _lock:
        if p not in cache:
            if (p, count) not in _LIBS:
                raise ValueError(f"no oracle build over p = {p}")
            build()
            L = ctypes.CDLL(_LIBS[(p, count)])
            configure(L)
            assert L.orc_prime() == p and L.orc_counts_ops() == int(count)
            cache[p] = L
    return cache[p]


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
def encT(code: dict, w, p: int = P, _count: bool = False) -> np.ndarray:
    """G^T w for w in F^k (App. B, linear-time encoding)."""
    k, r = code["k"], code["r"]
    w = _u32(w)
    assert w.shape == (k,)
    c = _code_args(code)
    out = np.empty(k * r, dtype=np.uint32)
    lib(p, _count).orc_encT(k, r, *[_p(a) for a in c], _p(w), _p(out))
    return out


def syn(code: dict, v, p: int = P, _count: bool = False) -> np.ndarray:
    """G v for v in F^N (App. B, syndrome by the transposition principle)."""
    k, r = code["k"], code["r"]
    v = _u32(v)
    assert v.shape == (k * r,)
    c = _code_args(code)
    out = np.empty(k, dtype=np.uint32)
    lib(p, _count).orc_syn(k, r, *[_p(a) for a in c], _p(v), _p(out))
    return out


def field_ops(name: str, *args, p: int = P) -> int:
    """Field operations the oracle performs in one call of ``name`` ("encT" or
    "syn") with these arguments, counted by the counting build."""
    fn = {"encT": encT, "syn": syn}[name]
    L = lib(p, True)
    with _count_lock:
        L.orc_ops_reset()
        fn(*args, p=p, _count=True)
        return int(L.orc_ops_count())


# ---------------------------------------------------------------------------
# Protocol pvMVMD
# ---------------------------------------------------------------------------
def server_eval(W, Xhat, rows=None, p: int = P, nthreads: int = 1) -> np.ndarray:
    """Yhat = W Xhat mod p; W int8 m x n, Xhat uint32 B x n -> uint32 B x m.

    ``rows`` = (row0, row1) restricts the computation to a row range (other
    entries of the result are left zero).  ``nthreads`` > 1 splits the rows
    into blocks computed by that many host threads (the same per-entry sums).
    """
    W = np.ascontiguousarray(W, dtype=np.int8)
    Xhat = _u32(np.atleast_2d(Xhat))
    m, n = W.shape
    B = Xhat.shape[0]
    assert Xhat.shape == (B, n)
    Y = np.zeros((B, m), dtype=np.uint32)
    r0, r1 = (0, m) if rows is None else (int(rows[0]), min(m, int(rows[1])))
    L = lib(p)
    ranges = [(r0 + a, r0 + b) for a, b in _blocks(r1 - r0, nthreads, 8)]
    _run_blocks(lambda a, b: L.orc_server_eval_rows(_p(W, ctypes.c_int8), m, n, _p(Xhat), B, _p(Y), a, b),
                ranges, nthreads)
    return Y


def keygen(W, cx: dict, cy: dict, want_P: bool = True, want_Q: bool = True, p: int = P, nthreads: int = 1):
    """Preprocess: returns (PT, Q) with PT = (W Gx)^T (Nx x m), Q = Gy^T W (Ny x n).
    ``nthreads`` > 1: the row encodings (PT) and the column encodings (Q) are
    split into blocks computed by that many host threads."""
    W = np.ascontiguousarray(W, dtype=np.int8)
    m, n = W.shape
    assert cx["k"] == n and cy["k"] == m
    PT = np.empty((cx["N"], m), dtype=np.uint32) if want_P else None
    Q = np.empty((cy["N"], n), dtype=np.uint32) if want_Q else None
    cxa, cya = _code_args(cx), _code_args(cy)  # kept alive while the pointers are used
    ax = [_p(a) for a in cxa]
    ay = [_p(a) for a in cya]
    L = lib(p)
    if nthreads <= 1:
        L.orc_keygen(_p(W, ctypes.c_int8), m, n, cx["r"], *ax, cy["r"], *ay, _p(PT), _p(Q))
        return PT, Q
    if want_P:
        _run_blocks(lambda a, b: L.orc_keygen_PT_rows(_p(W, ctypes.c_int8), m, n, cx["r"], *ax, _p(PT), a, b),
                    _blocks(m, nthreads), nthreads)
    if want_Q:
        _run_blocks(lambda a, b: L.orc_keygen_Q_cols(_p(W, ctypes.c_int8), m, n, cy["r"], *ay, _p(Q), a, b),
                    _blocks(n, nthreads), nthreads)
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


def decode(PT, Yhat, ex_idx, ex_val, p: int = P, nthreads: int = 1) -> np.ndarray:
    """Decrypt: Y = Yhat - P e_x.  ``nthreads`` > 1: the columns are split over
    that many host threads."""
    PT = _u32(PT)
    Yhat = _u32(np.atleast_2d(Yhat))
    B, m = Yhat.shape
    assert PT.shape[1] == m
    ex_idx = _u32(ex_idx)
    ex_val = _u32(ex_val)
    tx = ex_idx.shape[1]
    assert ex_idx.shape == (B, tx) and ex_val.shape == (B, tx)
    assert int(ex_idx.max(initial=0)) < PT.shape[0]
    Y = np.empty_like(Yhat)
    L = lib(p)
    _run_blocks(lambda a, b: L.orc_decode(_p(PT), m, _p(Yhat[a:b]), b - a, _p(ex_idx[a:b]), _p(ex_val[a:b]), tx,
                                          _p(Y[a:b])), _blocks(B, nthreads), nthreads)
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
# Seeded sampling of the method's random draws (a written specification; see
# the comment above orc_sample_code in mvk_oracle.c)
# ---------------------------------------------------------------------------
# Domain-separation tags: ASCII "mvk-codx", "mvk-cody", "mvk-nois", "mvk-chal"
# read as big-endian 64-bit integers.
TAG_CODE_X = int.from_bytes(b"mvk-codx", "big")
TAG_CODE_Y = int.from_bytes(b"mvk-cody", "big")
TAG_NOISE = int.from_bytes(b"mvk-nois", "big")
TAG_CHALLENGE = int.from_bytes(b"mvk-chal", "big")


def sample_code(k: int, r: int, seed: int, tag: int, p: int = P) -> dict:
    """A random RAA code (App. B) drawn from (seed, tag): dict(k, r, N, pi1, pi2, v1, v2)."""
    N = int(k) * int(r)
    arrs = [np.empty(N, dtype=np.uint32) for _ in range(4)]
    lib(p).orc_sample_code(k, r, seed & (2**64 - 1), tag, *[_p(a) for a in arrs])
    return dict(k=int(k), r=int(r), N=N, pi1=arrs[0], pi2=arrs[1], v1=arrs[2], v2=arrs[3])


def sm64_draws(state: int, count: int, p: int = P) -> list:
    """The first ``count`` outputs of the generator started at ``state``."""
    out = (ctypes.c_uint64 * count)()
    lib(p).orc_sm64_draws(state & (2**64 - 1), count, out)
    return list(out)


def sample_sparse(count: int, N: int, t: int, seed: int, tag: int, p: int = P):
    """``count`` draws from E_t^N (Sec. 3) from (seed, tag): (idx, val), each count x t."""
    if t > N:
        raise ValueError("sparsity t exceeds length N")
    idx = np.empty((count, t), dtype=np.uint32)
    val = np.empty((count, t), dtype=np.uint32)
    lib(p).orc_sample_sparse(count, N, t, seed & (2**64 - 1), tag, _p(idx), _p(val))
    return idx, val


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
