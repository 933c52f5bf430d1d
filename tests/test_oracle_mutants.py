"""The oracle's pins catch plausible mistakes: each test below plants one
mistake in a copy of the oracle's C source (a dropped term, a wrong index,
sign or orientation, a transposed operand), builds it with gcc into a
temporary directory, and checks that at least one pin of a battery (the same
independent routes as tests/test_oracle_pins.py: dense factor matrices of
App. B, Python big integers, closed forms, completeness and tamper rejection)
fails on it, while the unmodified oracle passes them all.  CPU only."""
import contextlib
import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle
import synth
from tests.test_oracle_pins import _matmul, brute_server, dense_G, matvec, transpose

P = synth.P
SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "mvk_oracle.c")

# (name, text in mvk_oracle.c, replacement): each text occurs exactly once
MUTANTS = [
    ("encT drops V1", "for (uint64_t j = 0; j < N; j++) t1[j] = fmul(v1[j], t1[j]);", ";"),
    ("encT second accumulation as a suffix sum",
     "for (uint64_t j = 1; j < N; j++) t0[j] = fadd(t0[j - 1], t0[j]);",
     "for (uint64_t j = N - 1; j-- > 0;) t0[j] = fadd(t0[j], t0[j + 1]);"),
    ("encT repeats interleaved instead of in blocks", "t0[j] = w[j / r];", "t0[j] = w[j % k];"),
    ("syn scatters Pi2 as a gather", "for (uint64_t j = 0; j < N; j++) s1[pi2[j]] = s0[j];",
     "for (uint64_t j = 0; j < N; j++) s1[j] = s0[pi2[j]];"),
    ("syn drops V2", "for (uint64_t j = 0; j < N; j++) s0[j] = fmul(v2[j], s0[j]);", ";"),
    ("syn folds with a wrong stride", "acc = fadd(acc, s0[i * r + q]);", "acc = fadd(acc, s0[q * k + i]);"),
    ("server reads int8 weights as unsigned", "fmul(emb(w[k]), x[k])", "fmul((uint8_t)w[k], x[k])"),
    ("keygen encodes W transposed for Q", "col[i] = (uint32_t)emb(W[(uint64_t)i * n + k]);",
     "col[i] = (uint32_t)emb(W[(uint64_t)k * m + i]);"),
    ("encode subtracts the mask", "Xhat[(uint64_t)b * n + k] = (uint32_t)fadd(X[(uint64_t)b * n + k], xp[k]);",
     "Xhat[(uint64_t)b * n + k] = (uint32_t)fsub(X[(uint64_t)b * n + k], xp[k]);"),
    ("decode adds the mask", "(uint32_t)fsub(Yhat[(uint64_t)b * m + i], mask);",
     "(uint32_t)fadd(Yhat[(uint64_t)b * m + i], mask);"),
    ("verify drops the challenge weights in u",
     "u[k] = fadd(u[k], fmul(ev[s], Q[(uint64_t)ei[s] * n + k]));",
     "u[k] = fadd(u[k], Q[(uint64_t)ei[s] * n + k]);"),
    ("verify never rejects", "if (l != rr) accept[b] = 0;", "if (0) accept[b] = 0;"),
]


@contextlib.contextmanager
def mutant(tmp_path, name, text, repl):
    src = open(SRC).read()
    assert src.count(text) == 1, name
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(text, repl))
    so = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", "-O1", "-std=c99", "-fPIC", "-shared", f"-DORC_P={P}ULL", "-o", str(so), str(path)])
    L = ctypes.CDLL(str(so))
    oracle.configure(L)
    saved = oracle.lib(P)
    oracle._lib[P] = L
    try:
        yield
    finally:
        oracle._lib[P] = saved


def _instance(cid, m, n, B, r, tx, ty=31, ell=2):
    W = synth.weights(synth.seed_for(cid, 1), m, n)
    X = synth.field_uniform(synth.seed_for(cid, 2), (B, n))
    cx = synth.raa_code(synth.seed_for(cid, 3), n, r)
    cy = synth.raa_code(synth.seed_for(cid, 4), m, r)
    exi, exv = synth.sparse(synth.seed_for(cid, 5), B, cx["N"], tx)
    eyi, eyv = synth.sparse(synth.seed_for(cid, 6), ell, cy["N"], ty)
    return W, X, cx, cy, exi, exv, eyi, eyv


def battery() -> dict:
    """Pin name -> passed."""
    out = {}
    code = synth.raa_code(123, 5, 3)
    G = dense_G(code, P)
    w = synth.field_uniform(1, 5)
    v = synth.field_uniform(2, 15)
    out["encT = dense G^T w"] = oracle.encT(code, w).tolist() == matvec(transpose(G), w, P)
    out["syn = dense G v"] = oracle.syn(code, v).tolist() == matvec(G, v, P)
    ident = synth.identity_code(9, 1)
    e0 = np.zeros(9, dtype=np.uint32)
    e0[0] = 1
    out["encT closed form"] = oracle.encT(ident, e0).tolist() == [j + 1 for j in range(9)]
    Wt = synth.weights(7, 6, 11, lo=-128, hi=127)
    Xt = synth.field_uniform(8, (2, 11))
    out["server = big integers"] = oracle.server_eval(Wt, Xt).tolist() == brute_server(Wt, Xt, P)
    Wk = synth.weights(31, 5, 4)
    cx, cy = synth.raa_code(32, 4, 3), synth.raa_code(33, 5, 2)
    PT, Q = oracle.keygen(Wk, cx, cy)
    Wf = [[int(x) % P for x in row] for row in Wk]
    out["keygen = dense"] = (PT.tolist() == transpose(_matmul(Wf, dense_G(cx, P), P))
                             and Q.tolist() == _matmul(transpose(dense_G(cy, P)), Wf, P))
    W, X, cx, cy, exi, exv, eyi, eyv = _instance(940, 40, 30, 2, 3, 6)
    PT, Q = oracle.keygen(W, cx, cy)
    Xh = oracle.encode(cx, X, exi, exv)
    Yh = oracle.server_eval(W, Xh)
    acc, _, _ = oracle.verify(cy, Q, Xh, Yh, eyi, eyv)
    out["completeness: accepted"] = bool(acc.all())
    out["completeness: decrypts to W x"] = oracle.decode(PT, Yh, exi, exv).tolist() == brute_server(W, X, P)
    bad = Yh.copy()
    bad[1, 5] = (int(bad[1, 5]) + 3) % P
    acc, _, _ = oracle.verify(cy, Q, Xh, bad, eyi, eyv)
    out["tamper rejected"] = acc.tolist() == [True, False]
    return out


def test_unmodified_oracle_passes_the_battery():
    res = battery()
    assert all(res.values()), [k for k, ok in res.items() if not ok]


@pytest.mark.parametrize("name,text,repl", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_fails_a_pin(tmp_path, name, text, repl):
    with mutant(tmp_path, name, text, repl):
        try:
            res = battery()
        except Exception as e:  # a crash is also a failed pin
            res = {"raised " + type(e).__name__: False}
    assert not all(res.values()), f"{name}: every pin still passes"
