"""Pins of the CPU oracle against facts the paper and mathematics fix.

None of these tests re-types the oracle's own formulas: each compares the
oracle with an independent route (dense factor matrices of App. B, Python
big-integer arithmetic, closed forms, algebraic identities, exact
probabilities from Lemma 5.1, the parameter values printed in Sec. 7.1).
"""
import functools
import math
import os

import numpy as np
import pytest

import oracle
import synth

P = synth.P
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


class Fp:
    """The oracle and the field-dependent draws bound to one prime p."""

    DRAWS = ("field_uniform", "field_nonzero", "raa_code", "sparse", "tamper_delta")

    def __init__(self, p):
        self.p = p

    def __getattr__(self, name):
        f = getattr(synth, name) if name in self.DRAWS else getattr(oracle, name)
        return functools.partial(f, p=self.p)


@pytest.fixture(params=[synth.P, synth.P_BABYBEAR], ids=["m31", "babybear"])
def p(request):
    return request.param


# ---------------------------------------------------------------------------
# Dense construction of G_RAA from the element-wise definitions of App. B.
# 1-based (i, j) as printed; Python integers, reduction only at the end.
# ---------------------------------------------------------------------------
def _mat(rows, cols, f):
    return [[f(i, j) for j in range(1, cols + 1)] for i in range(1, rows + 1)]


def _matmul(A, B, p):
    n, k, m = len(A), len(B), len(B[0])
    return [[sum(A[i][t] * B[t][j] for t in range(k)) % p for j in range(m)] for i in range(n)]


def dense_G(code, p):
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
        G = _matmul(G, F, p)
    return G  # k x N


def matvec(M, v, p):
    return [sum(int(a) * int(b) for a, b in zip(row, v)) % p for row in M]


def transpose(M):
    return [list(c) for c in zip(*M)]


CODE_SHAPES = [(3, 2), (4, 3), (5, 4), (6, 1), (2, 5)]


@pytest.mark.parametrize("k,r", CODE_SHAPES)
def test_encT_and_syn_match_dense_factor_product(k, r, p):
    o = Fp(p)
    code = o.raa_code(100 + 10 * k + r, k, r)
    G = dense_G(code, p)
    GT = transpose(G)
    for s in range(3):
        w = o.field_uniform(7000 + s, k)
        v = o.field_uniform(8000 + s, k * r)
        assert o.encT(code, w).tolist() == matvec(GT, w, p)
        assert o.syn(code, v).tolist() == matvec(G, v, p)


def test_dense_G_with_small_values_by_hand(p):
    o = Fp(p)
    # k=2, r=2, identity permutations, unit diagonals: G = R A A with
    # R = [[1,1,0,0],[0,0,1,1]] and (A A)_{ij} = j - i + 1 for i <= j.
    code = synth.identity_code(2, 2)
    # G^T w for w = (1, 0): repeat -> (1,1,0,0); prefix -> (1,2,2,2); prefix -> (1,3,5,7)
    assert o.encT(code, [1, 0]).tolist() == [1, 3, 5, 7]
    # w = (0, 1): repeat -> (0,0,1,1); prefix -> (0,0,1,2); prefix -> (0,0,1,3)
    assert o.encT(code, [0, 1]).tolist() == [0, 0, 1, 3]
    # G v for v = e_0 (first unit vector): suffix -> (1,0,0,0); suffix -> (1,0,0,0);
    # fold -> (1, 0).  v = e_3: suffix -> (1,1,1,1); suffix -> (4,3,2,1); fold -> (7, 3).
    assert o.syn(code, [1, 0, 0, 0]).tolist() == [1, 0]
    assert o.syn(code, [0, 0, 0, 1]).tolist() == [7, 3]


@pytest.mark.parametrize("N", [1, 2, 7, 64, 1000])
def test_closed_forms_identity_code(N, p):
    o = Fp(p)
    code = synth.identity_code(N, 1)
    e0 = np.zeros(N, dtype=np.uint32)
    e0[0] = 1
    # two prefix sums of the first unit vector: j + 1
    assert o.encT(code, e0).tolist() == [j + 1 for j in range(N)]
    eN = np.zeros(N, dtype=np.uint32)
    eN[N - 1] = 1
    # two suffix sums of the last unit vector: N - i
    assert o.syn(code, eN).tolist() == [N - i for i in range(N)]


@pytest.mark.parametrize("k,r", [(16, 3), (100, 2), (37, 4)])
def test_linearity(k, r, p):
    o = Fp(p)
    code = o.raa_code(555 + k, k, r)
    x = o.field_uniform(1, k)
    y = o.field_uniform(2, k)
    a = 1234567891
    lhs = o.encT(code, (a * x.astype(object) + y.astype(object)) % p)
    rhs = (a * o.encT(code, x).astype(object) + o.encT(code, y).astype(object)) % p
    assert lhs.tolist() == rhs.tolist()
    u = o.field_uniform(3, k * r)
    v = o.field_uniform(4, k * r)
    lhs = o.syn(code, (a * u.astype(object) + v.astype(object)) % p)
    rhs = (a * o.syn(code, u).astype(object) + o.syn(code, v).astype(object)) % p
    assert lhs.tolist() == rhs.tolist()


@pytest.mark.parametrize("k,r", [(16, 3), (257, 2), (50, 4)])
def test_transposition_identity(k, r, p):
    """e^T (G^T y) = (G e)^T y for every e, y (App. B, transposition principle)."""
    o = Fp(p)
    code = o.raa_code(999 + k, k, r)
    for s in range(3):
        y = o.field_uniform(10 + s, k)
        e = o.field_uniform(20 + s, k * r)
        lhs = sum(int(a) * int(b) for a, b in zip(e, o.encT(code, y))) % p
        rhs = sum(int(a) * int(b) for a, b in zip(o.syn(code, e), y)) % p
        assert lhs == rhs


@pytest.mark.parametrize("k,r", [(1, 1), (7, 3), (100, 2), (257, 8)])
def test_raa_cost_within_the_bounds_of_app_b(k, r, p):
    """App. B: an encoding costs at most 4N field operations (two diagonal
    scalings and two prefix sums), a syndrome at most 5N (plus the fold)."""
    o = Fp(p)
    code = o.raa_code(2000 + k, k, r)
    N = k * r
    w = o.field_uniform(1, k)
    v = o.field_uniform(2, N)
    enc_ops = oracle.field_ops("encT", code, w, p=p)
    syn_ops = oracle.field_ops("syn", code, v, p=p)
    assert 0 < enc_ops <= 4 * N
    assert 0 < syn_ops <= 5 * N
    # the counting build computes the same values as the build the tests use
    assert np.array_equal(oracle.encT(code, w, p=p, _count=True), o.encT(code, w))


def test_masks_look_uniform(p):
    """Privacy sanity check (the mask's pseudorandomness is the dual-LPN
    assumption, not something a test can prove): the masks Gx e of sparse noise
    are nonzero almost everywhere and spread evenly over F_p (chi-square over
    16 buckets, 8 masks of 4096 entries)."""
    o = Fp(p)
    n, r, t = 4096, 3, 64
    code = o.raa_code(3000, n, r)
    idx, val = o.sparse(3001, 8, n * r, t)
    masks = o.encode(code, np.zeros((8, n), dtype=np.uint32), idx, val)
    assert (masks != 0).mean() > 0.999
    counts = np.bincount((masks.astype(np.uint64) * 16 // p).ravel().astype(np.int64), minlength=16)
    expect = masks.size / 16
    chi2 = float(((counts - expect) ** 2 / expect).sum())
    assert chi2 < 37.7  # 15 degrees of freedom, p = 0.001


# ---------------------------------------------------------------------------
# Server evaluation against Python big integers
# ---------------------------------------------------------------------------
def brute_server(W, X, p):
    W = [[int(v) for v in row] for row in W]
    out = []
    for x in np.atleast_2d(X):
        xs = [int(v) for v in x]
        out.append([sum(w * xv for w, xv in zip(row, xs)) % p for row in W])
    return out


@pytest.mark.parametrize("m,n,B", [(1, 1, 1), (3, 5, 2), (17, 33, 3), (64, 40, 1)])
def test_server_eval_brute_force(m, n, B, p):
    o = Fp(p)
    W = synth.weights(m * 7 + n, m, n, lo=-128, hi=127)
    X = o.field_uniform(m + 3 * n, (B, n))
    assert o.server_eval(W, X).tolist() == brute_server(W, X, p)


def test_server_eval_extremes(p):
    o = Fp(p)
    n = 300
    for wv in (-128, -127, 127):
        W = np.full((4, n), wv, dtype=np.int8)
        X = np.full((2, n), p - 1, dtype=np.uint32)
        X[1, ::2] = 0
        assert o.server_eval(W, X).tolist() == brute_server(W, X, p)


def test_server_eval_closed_forms(p):
    o = Fp(p)
    n = 50
    X = o.field_uniform(77, (2, n))
    I = np.eye(n, dtype=np.int8)
    assert np.array_equal(o.server_eval(I, X), X)
    M = np.full((3, n), -1, dtype=np.int8)
    want = [[(-sum(int(v) for v in x)) % p] * 3 for x in X]
    assert o.server_eval(M, X).tolist() == want


def test_server_eval_row_range(p):
    o = Fp(p)
    W = synth.weights(5, 20, 9)
    X = o.field_uniform(6, (2, 9))
    full = o.server_eval(W, X)
    part = o.server_eval(W, X, rows=(4, 11))
    assert np.array_equal(part[:, 4:11], full[:, 4:11])
    assert not part[:, :4].any() and not part[:, 11:].any()


# ---------------------------------------------------------------------------
# Preprocess against dense G
# ---------------------------------------------------------------------------
def test_keygen_against_dense(p):
    o = Fp(p)
    m, n, rx, ry = 5, 4, 3, 2
    W = synth.weights(31, m, n)
    cx = o.raa_code(32, n, rx)
    cy = o.raa_code(33, m, ry)
    PT, Q = o.keygen(W, cx, cy)
    Wf = [[int(v) % p for v in row] for row in W]
    Gx = dense_G(cx, p)  # n x Nx
    Gy = dense_G(cy, p)  # m x Ny
    Pm = _matmul(Wf, Gx, p)  # m x Nx
    Qm = _matmul(transpose(Gy), Wf, p)  # Ny x n
    assert PT.tolist() == transpose(Pm)
    assert Q.tolist() == Qm


# ---------------------------------------------------------------------------
# Protocol completeness / soundness
# ---------------------------------------------------------------------------
def _instance(o, cid, m, n, B, r, tx, ty, ell):
    W = synth.weights(synth.seed_for(cid, 1), m, n)
    X = o.field_uniform(synth.seed_for(cid, 2), (B, n))
    cx = o.raa_code(synth.seed_for(cid, 3), n, r)
    cy = o.raa_code(synth.seed_for(cid, 4), m, r)
    exi, exv = o.sparse(synth.seed_for(cid, 5), B, cx["N"], tx)
    eyi, eyv = o.sparse(synth.seed_for(cid, 6), ell, cy["N"], ty)
    return W, X, cx, cy, exi, exv, eyi, eyv


@pytest.mark.parametrize("m,n,B,r,tx", [(256, 256, 1, 2, 8), (33, 70, 3, 3, 5), (8, 8, 2, 1, 3)])
def test_completeness(m, n, B, r, tx, p):
    o = Fp(p)
    W, X, cx, cy, exi, exv, eyi, eyv = _instance(o, 900 + m, m, n, B, r, tx, 31 if r * m >= 31 else 4, 2)
    PT, Q = o.keygen(W, cx, cy)
    Xh = o.encode(cx, X, exi, exv)
    Yh = o.server_eval(W, Xh)
    acc, vL, vR = o.verify(cy, Q, Xh, Yh, eyi, eyv)
    assert acc.all() and np.array_equal(vL, vR)
    Y = o.decode(PT, Yh, exi, exv)
    assert Y.tolist() == brute_server(W, X, p)
    # the mask actually changes the query (all but rare coordinates)
    assert (Xh != X).mean() > 0.9


def test_tamper_rejected_and_error_survives_masking(p):
    o = Fp(p)
    m, n, B = 64, 48, 2
    W, X, cx, cy, exi, exv, eyi, eyv = _instance(o, 950, m, n, B, 3, 6, 31, 2)
    PT, Q = o.keygen(W, cx, cy)
    Xh = o.encode(cx, X, exi, exv)
    Yh = o.server_eval(W, Xh)
    pos, delta = o.tamper_delta(951, 40, m)
    for t in range(40):
        bad = Yh.copy()
        b = t % B
        bad[b, pos[t]] = (int(bad[b, pos[t]]) + int(delta[t])) % p
        eyi2, eyv2 = o.sparse(5000 + t, 2, cy["N"], 31)
        acc, _, _ = o.verify(cy, Q, Xh, bad, eyi2, eyv2)
        assert not acc[b] and acc[1 - b]
        # y - M x = y^ - M x^ (proof of Theorem 6.1): the decrypted error equals the injected one
        Y = o.decode(PT, bad, exi, exv)
        good = o.decode(PT, Yh, exi, exv)
        diff = (Y.astype(np.int64) - good.astype(np.int64)) % p
        assert diff[b, pos[t]] == delta[t] and np.count_nonzero(diff) == 1


def test_swapped_columns_and_wrong_code_rejected(p):
    o = Fp(p)
    m, n, B = 40, 40, 2
    W, X, cx, cy, exi, exv, eyi, eyv = _instance(o, 960, m, n, B, 3, 6, 31, 2)
    _, Q = o.keygen(W, cx, cy, want_P=False)
    Xh = o.encode(cx, X, exi, exv)
    Yh = o.server_eval(W, Xh)
    acc, _, _ = o.verify(cy, Q, Xh, Yh[::-1].copy(), eyi, eyv)
    assert not acc.any()
    other = o.raa_code(961, m, 3)
    _, Q2 = o.keygen(W, cx, other, want_P=False)
    acc, _, _ = o.verify(cy, Q2, Xh, Yh, eyi, eyv)
    assert not acc.any()


def test_challenge_known_forgery_is_accepted(p):
    """A server that knows the challenges before answering can forge (why they
    are sampled after the responses are fixed, Protocol Batch-vMVMD)."""
    o = Fp(p)
    m, n = 30, 20
    W, X, cx, cy, exi, exv, eyi, eyv = _instance(o, 970, m, n, 1, 3, 4, 5, 2)
    _, Q = o.keygen(W, cx, cy, want_P=False)
    Xh = o.encode(cx, X, exi, exv)
    Yh = o.server_eval(W, Xh)
    # rows r_q = G_y e_q; any Delta orthogonal to both is invisible to the check.
    rs = []
    for q in range(2):
        e = np.zeros(cy["N"], dtype=np.uint32)
        e[eyi[q]] = eyv[q]
        rs.append([int(v) for v in o.syn(cy, e)])
    # Delta supported on three coordinates: solve the 2x3 system by a cross product.
    a, b = rs[0][:3], rs[1][:3]
    d = [(a[1] * b[2] - a[2] * b[1]) % p, (a[2] * b[0] - a[0] * b[2]) % p, (a[0] * b[1] - a[1] * b[0]) % p]
    assert any(d)
    bad = Yh.copy()
    for i in range(3):
        bad[0, i] = (int(bad[0, i]) + d[i]) % p
    acc, _, _ = o.verify(cy, Q, Xh, bad, eyi, eyv)
    assert acc[0]
    eyi2, eyv2 = o.sparse(971, 2, cy["N"], 5)
    acc, _, _ = o.verify(cy, Q, Xh, bad, eyi2, eyv2)
    assert not acc[0]


@pytest.mark.parametrize("t", [1, 2])
def test_acceptance_probability_lemma(t, p):
    """Lemma 5.1: with e uniform in E_t^N and z = G^T Delta of weight w, the check
    accepts exactly when supp(e) misses supp(z) (up to 1/(p-1)), i.e. with
    probability C(N - w, t) / C(N, t).  A degenerate code (identity
    permutations, unit diagonals, r = 1) gives codewords of known weight:
    Delta = e_i encodes to a vector supported on positions >= i (w = N - i)."""
    o = Fp(p)
    N = 12
    i = 5
    code = synth.identity_code(N, 1)
    W = np.eye(N, dtype=np.int8)
    _, Q = o.keygen(W, code, code, want_P=False)
    Xh = o.field_uniform(1, (1, N))
    Yh = o.server_eval(W, Xh)
    bad = Yh.copy()
    bad[0, i] = (int(bad[0, i]) + 17) % p
    w = N - i
    assert np.count_nonzero(o.encT(code, (bad[0].astype(np.int64) - Yh[0]) % p)) == w
    trials = 6000
    eyi, eyv = o.sparse(4242 + t, trials, N, t)
    hits = 0
    for s in range(trials):
        acc, _, _ = o.verify(code, Q, Xh, bad, eyi[s:s + 1], eyv[s:s + 1])
        hits += int(acc[0])
    prob = math.comb(N - w, t) / math.comb(N, t)
    sd = math.sqrt(prob * (1 - prob) / trials)
    assert abs(hits / trials - prob) < 5 * sd + 1e-9


# ---------------------------------------------------------------------------
# Protocol Batch-vMVMD (Sec. 5.4)
# ---------------------------------------------------------------------------
def batch_instance(o, cid, m, n, B, r, r2, t, ell, t2, ell2):
    """B claims M_b x_b = y_b under one primary code; Q_b = G^T M_b."""
    Ws = [synth.weights(synth.seed_for(cid, synth.PURPOSE_W, b), m, n) for b in range(B)]
    X = o.field_uniform(synth.seed_for(cid, synth.PURPOSE_X), (B, n))
    cx = o.raa_code(synth.seed_for(cid, synth.PURPOSE_CX), n, 2)
    cy = o.raa_code(synth.seed_for(cid, synth.PURPOSE_CY), m, r)
    c2 = o.raa_code(synth.seed_for(cid, synth.PURPOSE_C2), B * n, r2)
    Qs = np.stack([o.keygen(W, cx, cy, want_P=False)[1] for W in Ws])
    Y = np.concatenate([o.server_eval(W, X[b:b + 1]) for b, W in enumerate(Ws)])
    ei, ev = o.sparse(synth.seed_for(cid, synth.PURPOSE_CHAL), ell, cy["N"], t)
    e2i, e2v = o.sparse(synth.seed_for(cid, synth.PURPOSE_CHAL2), ell2, c2["N"], t2)
    return Ws, X, Y, cy, c2, Qs, ei, ev, e2i, e2v


def test_batch_aux_against_dense(p):
    """Qaux = Qt^T G' with Qt = [Q_1 | ... | Q_B]^T and G' built densely."""
    o = Fp(p)
    Ws, X, Y, cy, c2, Qs, *_ = batch_instance(o, 980, 3, 2, 2, 2, 2, 1, 1, 1, 1)
    B, N, n = Qs.shape
    QtT = [[int(Qs[b, i, c]) for b in range(B) for c in range(n)] for i in range(N)]  # N x Bn
    want = _matmul(QtT, dense_G(c2, p), p)  # N x N'
    assert o.batch_aux(Qs, c2).tolist() == want


def test_batch_identity_with_dense_matrices(p):
    """Both sides of each secondary check against Python integers and dense
    matrices: sL = e^T (Qt^T G') e' and sR = (G' e')^T (Qt e); original
    sides vR = e^T (G^T y_b), vL = (Q_b^T e)^T x_b."""
    o = Fp(p)
    Ws, X, Y, cy, c2, Qs, ei, ev, e2i, e2v = batch_instance(o, 981, 4, 3, 2, 2, 2, 2, 2, 2, 2)
    B, N, n = Qs.shape
    Qaux = o.batch_aux(Qs, c2)
    ut = o.batch_project(Qs, ei, ev)
    acc, ok, vL, vR, sL, sR = o.batch_verify(cy, c2, Qaux, X, Y, ei, ev, ut, e2i, e2v)
    assert acc.all() and ok
    G2 = dense_G(c2, p)  # Bn x N'
    Gy = dense_G(cy, p)  # m x N
    QtT = [[int(Qs[b, i, c]) for b in range(B) for c in range(n)] for i in range(N)]
    for q in range(ei.shape[0]):
        e = [0] * N
        for j, v in zip(ei[q], ev[q]):
            e[int(j)] = int(v)
        u = matvec(transpose(QtT), e, p)  # Qt e, length Bn
        assert ut[q].tolist() == u
        for j in range(e2i.shape[0]):
            e2 = [0] * c2["N"]
            for c, v in zip(e2i[j], e2v[j]):
                e2[int(c)] = int(v)
            g = matvec(G2, e2, p)
            assert int(sR[q, j]) == sum(a * b for a, b in zip(g, u)) % p
            aux_e2 = matvec(_matmul(QtT, G2, p), e2, p)
            assert int(sL[q, j]) == sum(a * b for a, b in zip(e, aux_e2)) % p
        for b in range(B):
            z = matvec(transpose(Gy), [int(v) for v in Y[b]], p)
            assert int(vR[q, b]) == sum(a * b2 for a, b2 in zip(e, z)) % p
            assert int(vL[q, b]) == sum(int(a) * int(x) for a, x in zip(u[b * n:(b + 1) * n], X[b])) % p


def test_batch_completeness_and_rejections(p):
    o = Fp(p)
    m, n, B = 40, 24, 3
    Ws, X, Y, cy, c2, Qs, ei, ev, e2i, e2v = batch_instance(o, 982, m, n, B, 3, 2, 31, 2, 31, 2)
    Qaux = o.batch_aux(Qs, c2)
    ut = o.batch_project(Qs, ei, ev)
    acc, ok, *_ = o.batch_verify(cy, c2, Qaux, X, Y, ei, ev, ut, e2i, e2v)
    assert acc.all() and ok
    # a wrong claim: only that claim fails the original checks
    bad = Y.copy()
    bad[1, 7] = (int(bad[1, 7]) + 5) % p
    acc, ok, *_ = o.batch_verify(cy, c2, Qaux, X, bad, ei, ev, ut, e2i, e2v)
    assert acc.tolist() == [True, False, True] and ok
    # a wrong projection: the secondary checks reject the batch
    ut2 = ut.copy()
    ut2[0, 30] = (int(ut2[0, 30]) + 1) % p
    acc, ok, _, _, sL, sR = o.batch_verify(cy, c2, Qaux, X, Y, ei, ev, ut2, e2i, e2v)
    assert not ok and not acc.any() and (sL[0] != sR[0]).all() and (sL[1] == sR[1]).all()


def test_batch_consistent_forgery_caught_by_secondary_check(p):
    """The server sees the primary challenges (it computes Qt e).  It can change
    claim b's result by Delta and its projection u_b so that every original
    check passes; only the secondary check, drawn after, catches it."""
    o = Fp(p)
    m, n, B = 30, 16, 2
    Ws, X, Y, cy, c2, Qs, ei, ev, e2i, e2v = batch_instance(o, 983, m, n, B, 3, 2, 31, 2, 31, 2)
    Qaux = o.batch_aux(Qs, c2)
    ut = o.batch_project(Qs, ei, ev)
    bad = Y.copy()
    bad[0, 2] = (int(bad[0, 2]) + 1000) % p
    forged = ut.copy()
    x0 = [int(v) for v in X[0]]
    inv_x = pow(x0[0], p - 2, p)
    for q in range(ei.shape[0]):
        # the original check for claim 0 needs u_0 . x_0 to move by e^T G^T Delta
        e = np.zeros(cy["N"], dtype=np.uint32)
        e[ei[q]] = ev[q]
        shift = (1000 * int(o.syn(cy, e)[2])) % p
        forged[q, 0] = (int(forged[q, 0]) + shift * inv_x) % p
    acc, ok, vL, vR, _, _ = o.batch_verify(cy, c2, Qaux, X, bad, ei, ev, forged, e2i, e2v)
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
