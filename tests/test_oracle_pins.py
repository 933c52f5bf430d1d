"""Pins of the CPU oracle against facts the paper and mathematics fix.

None of these tests re-types the oracle's own formulas: each compares the
oracle with an independent route (dense factor matrices of App. B, Python
big-integer arithmetic, closed forms, algebraic identities, exact
probabilities from Lemma 5.1, the parameter values printed in Sec. 7.1).
"""
import math
import os

import numpy as np
import pytest

import oracle
import synth

P = synth.P
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# Dense construction of G_RAA from the element-wise definitions of App. B.
# 1-based (i, j) as printed; Python integers, reduction only at the end.
# ---------------------------------------------------------------------------
def _mat(rows, cols, f):
    return [[f(i, j) for j in range(1, cols + 1)] for i in range(1, rows + 1)]


def _matmul(A, B):
    n, k, m = len(A), len(B), len(B[0])
    return [[sum(A[i][t] * B[t][j] for t in range(k)) % P for j in range(m)] for i in range(n)]


def dense_G(code):
    k, r, N = code["k"], code["r"], code["N"]
    pi1 = [int(x) + 1 for x in code["pi1"]]  # 1-based pi(j)
    pi2 = [int(x) + 1 for x in code["pi2"]]
    v1 = [int(x) for x in code["v1"]]
    v2 = [int(x) for x in code["v2"]]
    R = _mat(k, N, lambda i, j: 1 if (i - 1) * r < j <= i * r else 0)
    Pi1 = _mat(N, N, lambda i, j: 1 if pi1[j - 1] == i else 0)
    Pi2 = _mat(N, N, lambda i, j: 1 if pi2[j - 1] == i else 0)
    V1 = _mat(N, N, lambda i, j: v1[i - 1] if i == j else 0)
    V2 = _mat(N, N, lambda i, j: v2[i - 1] if i == j else 0)
    A = _mat(N, N, lambda i, j: 1 if i <= j else 0)
    G = R
    for F in (Pi1, V1, A, Pi2, V2, A):
        G = _matmul(G, F)
    return G  # k x N


def matvec(M, v):
    return [sum(int(a) * int(b) for a, b in zip(row, v)) % P for row in M]


def transpose(M):
    return [list(c) for c in zip(*M)]


CODE_SHAPES = [(3, 2), (4, 3), (5, 4), (6, 1), (2, 5)]


@pytest.mark.parametrize("k,r", CODE_SHAPES)
def test_encT_and_syn_match_dense_factor_product(k, r):
    code = synth.raa_code(100 + 10 * k + r, k, r)
    G = dense_G(code)
    GT = transpose(G)
    for s in range(3):
        w = synth.field_uniform(7000 + s, k)
        v = synth.field_uniform(8000 + s, k * r)
        assert oracle.encT(code, w).tolist() == matvec(GT, w)
        assert oracle.syn(code, v).tolist() == matvec(G, v)


def test_dense_G_with_small_values_by_hand():
    # k=2, r=2, identity permutations, unit diagonals: G = R A A with
    # R = [[1,1,0,0],[0,0,1,1]] and (A A)_{ij} = j - i + 1 for i <= j.
    code = synth.identity_code(2, 2)
    # G^T w for w = (1, 0): repeat -> (1,1,0,0); prefix -> (1,2,2,2); prefix -> (1,3,5,7)
    assert oracle.encT(code, [1, 0]).tolist() == [1, 3, 5, 7]
    # w = (0, 1): repeat -> (0,0,1,1); prefix -> (0,0,1,2); prefix -> (0,0,1,3)
    assert oracle.encT(code, [0, 1]).tolist() == [0, 0, 1, 3]
    # G v for v = e_0 (first unit vector): suffix -> (1,0,0,0); suffix -> (1,0,0,0);
    # fold -> (1, 0).  v = e_3: suffix -> (1,1,1,1); suffix -> (4,3,2,1); fold -> (7, 3).
    assert oracle.syn(code, [1, 0, 0, 0]).tolist() == [1, 0]
    assert oracle.syn(code, [0, 0, 0, 1]).tolist() == [7, 3]


@pytest.mark.parametrize("N", [1, 2, 7, 64, 1000])
def test_closed_forms_identity_code(N):
    code = synth.identity_code(N, 1)
    e0 = np.zeros(N, dtype=np.uint32)
    e0[0] = 1
    # two prefix sums of the first unit vector: j + 1
    assert oracle.encT(code, e0).tolist() == [j + 1 for j in range(N)]
    eN = np.zeros(N, dtype=np.uint32)
    eN[N - 1] = 1
    # two suffix sums of the last unit vector: N - i
    assert oracle.syn(code, eN).tolist() == [N - i for i in range(N)]


@pytest.mark.parametrize("k,r", [(16, 3), (100, 2), (37, 4)])
def test_linearity(k, r):
    code = synth.raa_code(555 + k, k, r)
    x = synth.field_uniform(1, k)
    y = synth.field_uniform(2, k)
    a = 1234567891
    lhs = oracle.encT(code, (a * x.astype(object) + y.astype(object)) % P)
    rhs = (a * oracle.encT(code, x).astype(object) + oracle.encT(code, y).astype(object)) % P
    assert lhs.tolist() == rhs.tolist()
    u = synth.field_uniform(3, k * r)
    v = synth.field_uniform(4, k * r)
    lhs = oracle.syn(code, (a * u.astype(object) + v.astype(object)) % P)
    rhs = (a * oracle.syn(code, u).astype(object) + oracle.syn(code, v).astype(object)) % P
    assert lhs.tolist() == rhs.tolist()


@pytest.mark.parametrize("k,r", [(16, 3), (257, 2), (50, 4)])
def test_transposition_identity(k, r):
    """e^T (G^T y) = (G e)^T y for every e, y (App. B, transposition principle)."""
    code = synth.raa_code(999 + k, k, r)
    for s in range(3):
        y = synth.field_uniform(10 + s, k)
        e = synth.field_uniform(20 + s, k * r)
        lhs = sum(int(a) * int(b) for a, b in zip(e, oracle.encT(code, y))) % P
        rhs = sum(int(a) * int(b) for a, b in zip(oracle.syn(code, e), y)) % P
        assert lhs == rhs


# ---------------------------------------------------------------------------
# Server evaluation against Python big integers
# ---------------------------------------------------------------------------
def brute_server(W, X):
    W = [[int(v) for v in row] for row in W]
    out = []
    for x in np.atleast_2d(X):
        xs = [int(v) for v in x]
        out.append([sum(w * xv for w, xv in zip(row, xs)) % P for row in W])
    return out


@pytest.mark.parametrize("m,n,B", [(1, 1, 1), (3, 5, 2), (17, 33, 3), (64, 40, 1)])
def test_server_eval_brute_force(m, n, B):
    W = synth.weights(m * 7 + n, m, n, lo=-128, hi=127)
    X = synth.field_uniform(m + 3 * n, (B, n))
    assert oracle.server_eval(W, X).tolist() == brute_server(W, X)


def test_server_eval_extremes():
    n = 300
    for wv in (-128, -127, 127):
        W = np.full((4, n), wv, dtype=np.int8)
        X = np.full((2, n), P - 1, dtype=np.uint32)
        X[1, ::2] = 0
        assert oracle.server_eval(W, X).tolist() == brute_server(W, X)


def test_server_eval_closed_forms():
    n = 50
    X = synth.field_uniform(77, (2, n))
    I = np.eye(n, dtype=np.int8)
    assert np.array_equal(oracle.server_eval(I, X), X)
    M = np.full((3, n), -1, dtype=np.int8)
    want = [[(-sum(int(v) for v in x)) % P] * 3 for x in X]
    assert oracle.server_eval(M, X).tolist() == want


def test_server_eval_row_range():
    W = synth.weights(5, 20, 9)
    X = synth.field_uniform(6, (2, 9))
    full = oracle.server_eval(W, X)
    part = oracle.server_eval(W, X, rows=(4, 11))
    assert np.array_equal(part[:, 4:11], full[:, 4:11])
    assert not part[:, :4].any() and not part[:, 11:].any()


# ---------------------------------------------------------------------------
# Preprocess against dense G
# ---------------------------------------------------------------------------
def test_keygen_against_dense():
    m, n, rx, ry = 5, 4, 3, 2
    W = synth.weights(31, m, n)
    cx = synth.raa_code(32, n, rx)
    cy = synth.raa_code(33, m, ry)
    PT, Q = oracle.keygen(W, cx, cy)
    Wf = [[int(v) % P for v in row] for row in W]
    Gx = dense_G(cx)  # n x Nx
    Gy = dense_G(cy)  # m x Ny
    Pm = _matmul(Wf, Gx)  # m x Nx
    Qm = _matmul(transpose(Gy), Wf)  # Ny x n
    assert PT.tolist() == transpose(Pm)
    assert Q.tolist() == Qm


# ---------------------------------------------------------------------------
# Protocol completeness / soundness
# ---------------------------------------------------------------------------
def _instance(cid, m, n, B, r, tx, ty, ell):
    W = synth.weights(synth.seed_for(cid, 1), m, n)
    X = synth.field_uniform(synth.seed_for(cid, 2), (B, n))
    cx = synth.raa_code(synth.seed_for(cid, 3), n, r)
    cy = synth.raa_code(synth.seed_for(cid, 4), m, r)
    exi, exv = synth.sparse(synth.seed_for(cid, 5), B, cx["N"], tx)
    eyi, eyv = synth.sparse(synth.seed_for(cid, 6), ell, cy["N"], ty)
    return W, X, cx, cy, exi, exv, eyi, eyv


@pytest.mark.parametrize("m,n,B,r,tx", [(256, 256, 1, 2, 8), (33, 70, 3, 3, 5), (8, 8, 2, 1, 3)])
def test_completeness(m, n, B, r, tx):
    W, X, cx, cy, exi, exv, eyi, eyv = _instance(900 + m, m, n, B, r, tx, 31 if r * m >= 31 else 4, 2)
    PT, Q = oracle.keygen(W, cx, cy)
    Xh = oracle.encode(cx, X, exi, exv)
    Yh = oracle.server_eval(W, Xh)
    acc, vL, vR = oracle.verify(cy, Q, Xh, Yh, eyi, eyv)
    assert acc.all() and np.array_equal(vL, vR)
    Y = oracle.decode(PT, Yh, exi, exv)
    assert Y.tolist() == brute_server(W, X)
    # the mask actually changes the query (all but rare coordinates)
    assert (Xh != X).mean() > 0.9


def test_tamper_rejected_and_error_survives_masking():
    m, n, B = 64, 48, 2
    W, X, cx, cy, exi, exv, eyi, eyv = _instance(950, m, n, B, 3, 6, 31, 2)
    PT, Q = oracle.keygen(W, cx, cy)
    Xh = oracle.encode(cx, X, exi, exv)
    Yh = oracle.server_eval(W, Xh)
    pos, delta = synth.tamper_delta(951, 40, m)
    for t in range(40):
        bad = Yh.copy()
        b = t % B
        bad[b, pos[t]] = (int(bad[b, pos[t]]) + int(delta[t])) % P
        eyi2, eyv2 = synth.sparse(5000 + t, 2, cy["N"], 31)
        acc, _, _ = oracle.verify(cy, Q, Xh, bad, eyi2, eyv2)
        assert not acc[b] and acc[1 - b]
        # y - M x = y^ - M x^ (proof of Theorem 6.1): the decrypted error equals the injected one
        Y = oracle.decode(PT, bad, exi, exv)
        good = oracle.decode(PT, Yh, exi, exv)
        diff = (Y.astype(np.int64) - good.astype(np.int64)) % P
        assert diff[b, pos[t]] == delta[t] and np.count_nonzero(diff) == 1


def test_swapped_columns_and_wrong_code_rejected():
    m, n, B = 40, 40, 2
    W, X, cx, cy, exi, exv, eyi, eyv = _instance(960, m, n, B, 3, 6, 31, 2)
    _, Q = oracle.keygen(W, cx, cy, want_P=False)
    Xh = oracle.encode(cx, X, exi, exv)
    Yh = oracle.server_eval(W, Xh)
    acc, _, _ = oracle.verify(cy, Q, Xh, Yh[::-1].copy(), eyi, eyv)
    assert not acc.any()
    other = synth.raa_code(961, m, 3)
    _, Q2 = oracle.keygen(W, cx, other, want_P=False)
    acc, _, _ = oracle.verify(cy, Q2, Xh, Yh, eyi, eyv)
    assert not acc.any()


def test_challenge_known_forgery_is_accepted():
    """A server that knows the challenges before answering can forge (why they
    are sampled after the responses are fixed, Protocol Batch-vMVMD)."""
    m, n = 30, 20
    W, X, cx, cy, exi, exv, eyi, eyv = _instance(970, m, n, 1, 3, 4, 5, 2)
    _, Q = oracle.keygen(W, cx, cy, want_P=False)
    Xh = oracle.encode(cx, X, exi, exv)
    Yh = oracle.server_eval(W, Xh)
    # rows r_q = G_y e_q; any Delta orthogonal to both is invisible to the check.
    rs = []
    for q in range(2):
        e = np.zeros(cy["N"], dtype=np.uint32)
        e[eyi[q]] = eyv[q]
        rs.append([int(v) for v in oracle.syn(cy, e)])
    # Delta supported on three coordinates: solve the 2x3 system by a cross product.
    a, b = rs[0][:3], rs[1][:3]
    d = [(a[1] * b[2] - a[2] * b[1]) % P, (a[2] * b[0] - a[0] * b[2]) % P, (a[0] * b[1] - a[1] * b[0]) % P]
    assert any(d)
    bad = Yh.copy()
    for i in range(3):
        bad[0, i] = (int(bad[0, i]) + d[i]) % P
    acc, _, _ = oracle.verify(cy, Q, Xh, bad, eyi, eyv)
    assert acc[0]
    eyi2, eyv2 = synth.sparse(971, 2, cy["N"], 5)
    acc, _, _ = oracle.verify(cy, Q, Xh, bad, eyi2, eyv2)
    assert not acc[0]


@pytest.mark.parametrize("t", [1, 2])
def test_acceptance_probability_lemma(t):
    """Lemma 5.1: with e uniform in E_t^N and z = G^T Delta of weight w, the check
    accepts exactly when supp(e) misses supp(z) (up to 1/(p-1)), i.e. with
    probability C(N - w, t) / C(N, t).  A degenerate code (identity
    permutations, unit diagonals, r = 1) gives codewords of known weight:
    Delta = e_i encodes to a vector supported on positions >= i (w = N - i)."""
    N = 12
    i = 5
    code = synth.identity_code(N, 1)
    W = np.eye(N, dtype=np.int8)
    _, Q = oracle.keygen(W, code, code, want_P=False)
    Xh = synth.field_uniform(1, (1, N))
    Yh = oracle.server_eval(W, Xh)
    bad = Yh.copy()
    bad[0, i] = (int(bad[0, i]) + 17) % P
    w = N - i
    assert np.count_nonzero(oracle.encT(code, (bad[0].astype(np.int64) - Yh[0]) % P)) == w
    trials = 6000
    eyi, eyv = synth.sparse(4242 + t, trials, N, t)
    hits = 0
    for s in range(trials):
        acc, _, _ = oracle.verify(code, Q, Xh, bad, eyi[s:s + 1], eyv[s:s + 1])
        hits += int(acc[0])
    prob = math.comb(N - w, t) / math.comb(N, t)
    sd = math.sqrt(prob * (1 - prob) / trials)
    assert abs(hits / trials - prob) < 5 * sd + 1e-9


# ---------------------------------------------------------------------------
# Protocol Batch-vMVMD (Sec. 5.4)
# ---------------------------------------------------------------------------
def batch_instance(cid, m, n, B, r, r2, t, ell, t2, ell2):
    """B claims M_b x_b = y_b under one primary code; Q_b = G^T M_b."""
    Ws = [synth.weights(synth.seed_for(cid, synth.PURPOSE_W, b), m, n) for b in range(B)]
    X = synth.field_uniform(synth.seed_for(cid, synth.PURPOSE_X), (B, n))
    cx = synth.raa_code(synth.seed_for(cid, synth.PURPOSE_CX), n, 2)
    cy = synth.raa_code(synth.seed_for(cid, synth.PURPOSE_CY), m, r)
    c2 = synth.raa_code(synth.seed_for(cid, synth.PURPOSE_C2), B * n, r2)
    Qs = np.stack([oracle.keygen(W, cx, cy, want_P=False)[1] for W in Ws])
    Y = np.concatenate([oracle.server_eval(W, X[b:b + 1]) for b, W in enumerate(Ws)])
    ei, ev = synth.sparse(synth.seed_for(cid, synth.PURPOSE_CHAL), ell, cy["N"], t)
    e2i, e2v = synth.sparse(synth.seed_for(cid, synth.PURPOSE_CHAL2), ell2, c2["N"], t2)
    return Ws, X, Y, cy, c2, Qs, ei, ev, e2i, e2v


def test_batch_aux_against_dense():
    """Qaux = Qt^T G' with Qt = [Q_1 | ... | Q_B]^T and G' built densely."""
    Ws, X, Y, cy, c2, Qs, *_ = batch_instance(980, 3, 2, 2, 2, 2, 1, 1, 1, 1)
    B, N, n = Qs.shape
    QtT = [[int(Qs[b, i, c]) for b in range(B) for c in range(n)] for i in range(N)]  # N x Bn
    want = _matmul(QtT, dense_G(c2))  # N x N'
    assert oracle.batch_aux(Qs, c2).tolist() == want


def test_batch_identity_with_dense_matrices():
    """Both sides of each secondary check against Python integers and dense
    matrices: sL = e^T (Qt^T G') e' and sR = (G' e')^T (Qt e); original
    sides vR = e^T (G^T y_b), vL = (Q_b^T e)^T x_b."""
    Ws, X, Y, cy, c2, Qs, ei, ev, e2i, e2v = batch_instance(981, 4, 3, 2, 2, 2, 2, 2, 2, 2)
    B, N, n = Qs.shape
    Qaux = oracle.batch_aux(Qs, c2)
    ut = oracle.batch_project(Qs, ei, ev)
    acc, ok, vL, vR, sL, sR = oracle.batch_verify(cy, c2, Qaux, X, Y, ei, ev, ut, e2i, e2v)
    assert acc.all() and ok
    G2 = dense_G(c2)  # Bn x N'
    Gy = dense_G(cy)  # m x N
    QtT = [[int(Qs[b, i, c]) for b in range(B) for c in range(n)] for i in range(N)]
    for q in range(ei.shape[0]):
        e = [0] * N
        for j, v in zip(ei[q], ev[q]):
            e[int(j)] = int(v)
        u = matvec(transpose(QtT), e)  # Qt e, length Bn
        assert ut[q].tolist() == u
        for j in range(e2i.shape[0]):
            e2 = [0] * c2["N"]
            for c, v in zip(e2i[j], e2v[j]):
                e2[int(c)] = int(v)
            g = matvec(G2, e2)
            assert int(sR[q, j]) == sum(a * b for a, b in zip(g, u)) % P
            aux_e2 = matvec(_matmul(QtT, G2), e2)
            assert int(sL[q, j]) == sum(a * b for a, b in zip(e, aux_e2)) % P
        for b in range(B):
            z = matvec(transpose(Gy), [int(v) for v in Y[b]])
            assert int(vR[q, b]) == sum(a * b2 for a, b2 in zip(e, z)) % P
            assert int(vL[q, b]) == sum(int(a) * int(x) for a, x in zip(u[b * n:(b + 1) * n], X[b])) % P


def test_batch_completeness_and_rejections():
    m, n, B = 40, 24, 3
    Ws, X, Y, cy, c2, Qs, ei, ev, e2i, e2v = batch_instance(982, m, n, B, 3, 2, 31, 2, 31, 2)
    Qaux = oracle.batch_aux(Qs, c2)
    ut = oracle.batch_project(Qs, ei, ev)
    acc, ok, *_ = oracle.batch_verify(cy, c2, Qaux, X, Y, ei, ev, ut, e2i, e2v)
    assert acc.all() and ok
    # a wrong claim: only that claim fails the original checks
    bad = Y.copy()
    bad[1, 7] = (int(bad[1, 7]) + 5) % P
    acc, ok, *_ = oracle.batch_verify(cy, c2, Qaux, X, bad, ei, ev, ut, e2i, e2v)
    assert acc.tolist() == [True, False, True] and ok
    # a wrong projection: the secondary checks reject the batch
    ut2 = ut.copy()
    ut2[0, 30] = (int(ut2[0, 30]) + 1) % P
    acc, ok, _, _, sL, sR = oracle.batch_verify(cy, c2, Qaux, X, Y, ei, ev, ut2, e2i, e2v)
    assert not ok and not acc.any() and (sL[0] != sR[0]).all() and (sL[1] == sR[1]).all()


def test_batch_consistent_forgery_caught_by_secondary_check():
    """The server sees the primary challenges (it computes Qt e).  It can change
    claim b's result by Delta and its projection u_b so that every original
    check passes; only the secondary check, drawn after, catches it."""
    m, n, B = 30, 16, 2
    Ws, X, Y, cy, c2, Qs, ei, ev, e2i, e2v = batch_instance(983, m, n, B, 3, 2, 31, 2, 31, 2)
    Qaux = oracle.batch_aux(Qs, c2)
    ut = oracle.batch_project(Qs, ei, ev)
    bad = Y.copy()
    bad[0, 2] = (int(bad[0, 2]) + 1000) % P
    forged = ut.copy()
    x0 = [int(v) for v in X[0]]
    inv_x = pow(x0[0], P - 2, P)
    for q in range(ei.shape[0]):
        # the original check for claim 0 needs u_0 . x_0 to move by e^T G^T Delta
        e = np.zeros(cy["N"], dtype=np.uint32)
        e[ei[q]] = ev[q]
        shift = (1000 * int(oracle.syn(cy, e)[2])) % P
        forged[q, 0] = (int(forged[q, 0]) + shift * inv_x) % P
    acc, ok, vL, vR, _, _ = oracle.batch_verify(cy, c2, Qaux, X, bad, ei, ev, forged, e2i, e2v)
    assert (vL == vR).all()  # every original check passes
    assert not ok and not acc.any()


# ---------------------------------------------------------------------------
# Parameters printed in Sec. 7.1
# ---------------------------------------------------------------------------
def _golden_params():
    rows = {}
    with open(os.path.join(GOLDEN, "params_sec7_1.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                key, val = line.split("=")
                rows[key.strip()] = val.strip()
    return rows


def test_noise_weight_eq1_matches_printed_values():
    g = _golden_params()
    ns = [int(v) for v in g["n"].split(",")]
    txs = [int(v) for v in g["t_x"].split(",")]
    rate = int(g["inverse_rate"])
    for n, tx in zip(ns, txs):
        assert oracle.noise_weight(int(g["lambda"]), rate * n, float(g["delta"])) == tx


def test_verify_params_match_printed_values():
    g = _golden_params()
    q = int(g["q"])
    t, ell = oracle.verify_params(q, int(g["kappa"]), float(g["delta"]))
    assert (t, ell) == (int(g["t_y"]), int(g["ell"]))
    # the Mersenne field 2^31 - 1 gives the same pair
    assert oracle.verify_params(P, int(g["kappa"]), float(g["delta"])) == (31, 2)
    # a 64-bit field falls in the other case of the proof: one repetition
    assert oracle.verify_params(2**64 - 59, 40, 0.5) == (41, 1)
