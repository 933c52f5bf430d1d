"""GPU parity of the BabyBear build (libmvk_bb.so, p = 15 * 2^27 + 1, the field
of the paper's Sec. 7.1): every entry point against the oracle built over the
same field, bit-exact, on small and ragged shapes, at the exactness limit of
the server kernels, and on the Sec. 7.1 workload (n x n, r = 8, t_x of Eq. (1))."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import Instance, code, dev, host

pytestmark = pytest.mark.gpu
Q = synth.P_BABYBEAR


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_10264_amd as mvk  # noqa: F401  (raises if the library is missing)
    assert mvk._lib.load(Q).mvk_field_modulus() == Q


def _say(*a):
    print(*a, flush=True)


import paper_2609_10264_amd as mvk  # noqa: E402


def _dense(N, idx, val):
    e = np.zeros(N, dtype=np.uint32)
    e[idx] = val
    return e


# ---------------------------------------------------------------------------
# server_eval: every kernel family (one-query VALU, small-batch and streamed
# matrix-core kernels, packed weights)
# ---------------------------------------------------------------------------
SERVER_SHAPES = [
    (1, 1, 1), (17, 33, 2), (257, 4099, 1), (4096, 4096, 1), (100, 160, 5), (300, 1000, 16), (31, 2048, 64),
    (70, 999, 65), (16, 128, 130), (1000, 8192, 64), (257, 11008, 8), (64, 16448, 8), (129, 8192, 16),
    # packed, 17..32 queries and at least 192 blocks of 128 rows: the wide-tile kernel
    (24704, 520, 20),
]


@pytest.mark.parametrize("path", ["auto", "valu", "mfma", "packed"])
@pytest.mark.parametrize("m,n,B", SERVER_SHAPES)
def test_server_eval(m, n, B, path):
    _say(f"babybear server_eval m={m} n={n} B={B} path={path}")
    W = synth.weights(11 * m + n, m, n, lo=-128, hi=127)
    X = synth.field_uniform(13 * n + B, (B, n), p=Q)
    if path == "packed":
        got = mvk.server_eval(mvk.pack_weights(dev(W)), dev(X), p=Q)
    else:
        got = mvk.server_eval(dev(W), dev(X), path=path, p=Q)
    assert np.array_equal(host(got), oracle.server_eval(W, X, p=Q))


# centred representatives at both ends, a value whose balanced digits are all
# -128 but the top one, and 1
@pytest.mark.parametrize("path", ["valu", "mfma"])
@pytest.mark.parametrize("wv,xv", [(-128, Q - 8421504), (127, Q - 1), (-128, (Q - 1) // 2), (127, (Q + 1) // 2),
                                   (-127, 1)])
def test_server_eval_extremes(wv, xv, path):
    m, n = 5, mvk.MVK_MAX_N
    _say(f"babybear server_eval extreme w={wv} x={xv} path={path}")
    W = np.full((m, n), wv, dtype=np.int8)
    X = np.full((2, n), xv, dtype=np.uint32)
    X[1, ::3] = 0
    got = host(mvk.server_eval(dev(W), dev(X), path=path, p=Q))
    assert np.array_equal(got, oracle.server_eval(W, X, p=Q))


def test_server_eval_closed_form():
    n = 1000
    X = synth.field_uniform(5, (3, n), p=Q)
    M = np.full((7, n), -1, dtype=np.int8)
    want = np.array([[(-sum(int(v) for v in x)) % Q] * 7 for x in X], dtype=np.uint32)
    assert np.array_equal(host(mvk.server_eval(dev(M), dev(X), p=Q)), want)


# ---------------------------------------------------------------------------
# RAA encoding / syndrome (single-workgroup tiles and the segmented path)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("k,r,count", [(5, 2, 3), (1000, 3, 4), (4097, 4, 2), (6000, 4, 2), (16384, 1, 1),
                                         (2048, 8, 2), (1024, 8, 1), (2049, 8, 1), (700, 5, 65)])
def test_raa_encode_and_syndrome(k, r, count):
    _say(f"babybear raa k={k} r={r} count={count}")
    c = synth.raa_code(300 + k + r, k, r, p=Q)
    w = synth.field_uniform(301 + k, (count, k), p=Q)
    v = synth.field_uniform(302 + k, (count, k * r), p=Q)
    dc = code(c, Q)
    got_e = host(mvk.raa_encode(dc, dev(w)))
    got_s = host(mvk.raa_syndrome(dc, dev(v)))
    for i in range(count):
        assert np.array_equal(got_e[i], oracle.encT(c, w[i], p=Q))
        assert np.array_equal(got_s[i], oracle.syn(c, v[i], p=Q))


# ---------------------------------------------------------------------------
# Protocol pvMVMD end to end
# ---------------------------------------------------------------------------
SMALL = [  # cid, m, n, B, r, tx
    (0, 256, 256, 1, 2, 8),
    (50, 257, 130, 3, 3, 5),
    (51, 64, 1000, 2, 4, 17),
    (56, 1024, 1024, 1, 8, 160),   # the n = 2^10 point of Sec. 7.1
    (57, 700, 2049, 3, 8, 40),     # Nx = 16392: segmented noise syndromes
]


@pytest.mark.parametrize("cid,m,n,B,r,tx", SMALL)
def test_protocol(cid, m, n, B, r, tx):
    _say(f"babybear protocol cid={cid} m={m} n={n} B={B} r={r} tx={tx}")
    inst = Instance(cid, m, n, B, r, tx, p=Q).to_device()
    mvk.keygen(inst.key, inst.dW)
    PT, Qm = oracle.keygen(inst.W, inst.cx, inst.cy, p=Q)
    assert np.array_equal(host(inst.key.PT), PT)
    assert np.array_equal(host(inst.key.Q), Qm)
    dXh = mvk.encode(inst.key, inst.dX, inst.dexi, inst.dexv)
    Xh = oracle.encode(inst.cx, inst.X, inst.exi, inst.exv, p=Q)
    assert np.array_equal(host(dXh), Xh)
    dYh = mvk.server_eval(inst.dW, dXh, p=Q)
    Yh = oracle.server_eval(inst.W, Xh, p=Q)
    assert np.array_equal(host(dYh), Yh)
    ell = inst.eyi.shape[0]
    pos, delta = synth.tamper_delta(synth.seed_for(cid, synth.PURPOSE_TAMPER), B, m, p=Q)
    bad = Yh.copy()
    bad[B - 1, pos[0]] = (int(bad[B - 1, pos[0]]) + int(delta[0])) % Q
    for resp, want in ((Yh, [1] * B), (bad, [1] * (B - 1) + [0])):
        vL = torch.empty((ell, B), dtype=torch.int32, device="cuda")
        vR = torch.empty_like(vL)
        Y, acc, vL, vR = mvk.decode_verify(inst.key, dXh, dev(resp), inst.dexi, inst.dexv, inst.deyi, inst.deyv,
                                           vL=vL, vR=vR)
        oacc, ovL, ovR = oracle.verify(inst.cy, Qm, Xh, resp, inst.eyi, inst.eyv, p=Q)
        assert oacc.astype(np.uint32).tolist() == want == host(acc).tolist()
        assert np.array_equal(host(vL), ovL) and np.array_equal(host(vR), ovR)
        assert np.array_equal(host(Y), oracle.decode(PT, resp, inst.exi, inst.exv, p=Q))
    assert np.array_equal(host(Y)[:B - 1], oracle.server_eval(inst.W, inst.X, p=Q)[:B - 1])


@pytest.mark.parametrize("m,ry,B,ell", [(1000, 4, 2, 3), (2731, 3, 3, 5), (4096, 3, 2, 16), (5462, 3, 1, 2),
                                        (4096, 3, 9, 2), (2048, 8, 1, 2)])
def test_decode_verify_syndrome_shapes(m, ry, B, ell):
    _say(f"babybear decode_verify m={m} ry={ry} B={B} ell={ell}")
    inst = Instance(58, m, 64, B, 2, 9, ty=31, ell=ell, ry=ry, p=Q).to_device()
    mvk.keygen(inst.key, inst.dW)
    PT, Qm = oracle.keygen(inst.W, inst.cx, inst.cy, p=Q)
    dXh = mvk.encode(inst.key, inst.dX, inst.dexi, inst.dexv)
    Xh = host(dXh)
    Yh = oracle.server_eval(inst.W, Xh, p=Q)
    bad = Yh.copy()
    bad[0, m - 1] = (int(bad[0, m - 1]) + 1) % Q
    for resp, want in ((Yh, [1] * B), (bad, [0] + [1] * (B - 1))):
        vL = torch.empty((ell, B), dtype=torch.int32, device="cuda")
        vR = torch.empty_like(vL)
        Y, acc, vL, vR = mvk.decode_verify(inst.key, dXh, dev(resp), inst.dexi, inst.dexv, inst.deyi, inst.deyv,
                                           vL=vL, vR=vR)
        oacc, ovL, ovR = oracle.verify(inst.cy, Qm, Xh, resp, inst.eyi, inst.eyv, p=Q)
        assert oacc.astype(np.uint32).tolist() == want == host(acc).tolist()
        assert np.array_equal(host(vL), ovL) and np.array_equal(host(vR), ovR)
        assert np.array_equal(host(Y), oracle.decode(PT, resp, inst.exi, inst.exv, p=Q))


# ---------------------------------------------------------------------------
# Prepared (boost / pipelined standard mode) path and verification only
# ---------------------------------------------------------------------------
PREP = [  # cid, m, n, B, r_x, r_y, t_x, ell
    (80, 256, 256, 1, 2, 2, 8, 2),
    (81, 1000, 700, 3, 3, 2, 17, 3),
    (83, 300, 5500, 2, 3, 3, 64, 2),
    (86, 3000, 2000, 8, 2, 2, 16, 3),
    (87, 500, 400, 2, 2, 2, 9, 7),
    (89, 1024, 1024, 1, 8, 8, 160, 2),
    # one workgroup per column (4096-long columns) and the segment kernel
    # (ragged 4100 x 11008, five columns)
    (90, 4096, 3000, 8, 2, 2, 16, 2),
    (91, 4100, 11008, 5, 2, 2, 16, 2),
]


@pytest.mark.parametrize("cid,m,n,B,rx,ry,tx,ell", PREP)
def test_prepared_path(cid, m, n, B, rx, ry, tx, ell):
    _say(f"babybear prepared cid={cid} m={m} n={n} B={B}")
    inst = Instance(cid, m, n, B, rx, tx, ty=31, ell=ell, ry=ry, p=Q).to_device()
    mvk.keygen(inst.key, inst.dW)
    PT, Qm = oracle.keygen(inst.W, inst.cx, inst.cy, p=Q)
    prep = mvk.client_prepare(inst.key, inst.dexi, inst.dexv, inst.deyi, inst.deyv)
    Mx = oracle.encode(inst.cx, np.zeros((B, n), dtype=np.uint32), inst.exi, inst.exv, p=Q)
    assert np.array_equal(host(prep.Mx), Mx)
    assert np.array_equal(host(prep.My), oracle.server_eval(inst.W, Mx, p=Q))
    R = np.stack([oracle.syn(inst.cy, _dense(inst.cy["N"], inst.eyi[q], inst.eyv[q]), p=Q) for q in range(ell)])
    assert np.array_equal(host(prep.R), R)
    assert np.array_equal(host(prep.U), oracle.server_eval(np.ascontiguousarray(inst.W.T), R, p=Q))
    Xh = mvk.encode_masked(inst.key, inst.dX, prep)
    Xh_ref = oracle.encode(inst.cx, inst.X, inst.exi, inst.exv, p=Q)
    assert np.array_equal(host(Xh), Xh_ref)
    Yh = oracle.server_eval(inst.W, Xh_ref, p=Q)
    bad = Yh.copy()
    bad[B - 1, m // 2] = (int(bad[B - 1, m // 2]) + 12345) % Q
    for resp, want in ((Yh, [1] * B), (bad, [1] * (B - 1) + [0])):
        vL = torch.empty((ell, B), dtype=torch.int32, device="cuda")
        vR = torch.empty_like(vL)
        Y, acc, vL, vR = mvk.decode_verify_masked(inst.key, Xh, dev(resp), prep, vL=vL, vR=vR)
        oacc, ovL, ovR = oracle.verify(inst.cy, Qm, Xh_ref, resp, inst.eyi, inst.eyv, p=Q)
        assert oacc.astype(np.uint32).tolist() == want == host(acc).tolist()
        assert np.array_equal(host(vL), ovL) and np.array_equal(host(vR), ovR)
        assert np.array_equal(host(Y), oracle.decode(PT, resp, inst.exi, inst.exv, p=Q))


def test_client_turn():
    """decode_verify_encode_masked over BabyBear: the fused launch (4096 x
    4096, one column) and the two-launch form (3000 x 2000, eight columns)
    give the outputs of decode_verify_masked and encode_masked."""
    for cid, m, n, B in ((92, 4096, 4096, 1), (93, 3000, 2000, 8)):
        inst = Instance(cid, m, n, B, 3, 32, ty=31, ell=2, p=Q).to_device()
        mvk.keygen(inst.key, inst.dW)
        prep = mvk.client_prepare(inst.key, inst.dexi, inst.dexv, inst.deyi, inst.deyv)
        prep2 = mvk.client_prepare(inst.key, inst.dexi, inst.dexv, inst.deyi, inst.deyv)
        Xh = mvk.encode_masked(inst.key, inst.dX, prep)
        Yh = mvk.server_eval(inst.dW, Xh, p=Q)
        X2 = dev(synth.field_uniform(cid + 7, (B, n), p=Q))
        Y, acc, _, _, Xh2 = mvk.decode_verify_encode_masked(inst.key, Xh, Yh, prep, X2, prep2)
        Y1, acc1, _, _ = mvk.decode_verify_masked(inst.key, Xh, Yh, prep)
        assert torch.equal(Y, Y1) and torch.equal(acc, acc1) and host(acc).tolist() == [1] * B
        assert torch.equal(Xh2, mvk.encode_masked(inst.key, X2, prep2))


def test_verify_only():
    inst = Instance(59, 900, 500, 3, 3, 0, ell=2, p=Q).to_device()
    mvk.keygen(inst.key, inst.dW)
    _, Qm = oracle.keygen(inst.W, inst.cx, inst.cy, want_P=False, p=Q)
    Y = oracle.server_eval(inst.W, inst.X, p=Q)
    Y[1, 3] = (int(Y[1, 3]) + 1) % Q
    vL = torch.empty((2, 3), dtype=torch.int32, device="cuda")
    vR = torch.empty_like(vL)
    acc, vL, vR = mvk.verify(inst.key, inst.dX, dev(Y), inst.deyi, inst.deyv, vL=vL, vR=vR)
    oacc, ovL, ovR = oracle.verify(inst.cy, Qm, inst.X, Y, inst.eyi, inst.eyv, p=Q)
    assert host(acc).tolist() == oacc.astype(np.uint32).tolist() == [1, 0, 1]
    assert np.array_equal(host(vL), ovL) and np.array_equal(host(vR), ovR)


# ---------------------------------------------------------------------------
# Batch verification (Protocol Batch-vMVMD)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("cid,m,n,B,r,r2", [(100, 40, 24, 3, 3, 2), (102, 6000, 96, 2, 3, 2)])
def test_batch_verification(cid, m, n, B, r, r2):
    _say(f"babybear batch cid={cid} m={m} n={n} B={B}")
    sd = lambda purpose, sub=0: synth.seed_for(cid, purpose, sub)  # noqa: E731
    Ws = [synth.weights(sd(synth.PURPOSE_W, b), m, n) for b in range(B)]
    X = synth.field_uniform(sd(synth.PURPOSE_X), (B, n), p=Q)
    cx = synth.raa_code(sd(synth.PURPOSE_CX), n, 2, p=Q)
    cy = synth.raa_code(sd(synth.PURPOSE_CY), m, r, p=Q)
    c2 = synth.raa_code(sd(synth.PURPOSE_C2), B * n, r2, p=Q)
    Y = np.concatenate([oracle.server_eval(W, X[b:b + 1], p=Q) for b, W in enumerate(Ws)])
    ei, ev = synth.sparse(sd(synth.PURPOSE_CHAL), 2, cy["N"], 31, p=Q)
    e2i, e2v = synth.sparse(sd(synth.PURPOSE_CHAL2), 2, c2["N"], 31, p=Q)
    Qs = np.stack([oracle.keygen(W, cx, cy, want_P=False, p=Q)[1] for W in Ws])
    dcx, dcy, dc2 = code(cx, Q), code(cy, Q), code(c2, Q)
    keys = []
    for W in Ws:
        k = mvk.Key.allocate(m, n, dcx, dcy)
        mvk.keygen(k, dev(W))
        keys.append(k)
    QtT, Qaux = mvk.batch_preprocess([k.Q for k in keys], dc2)
    Qaux_ref = oracle.batch_aux(Qs, c2, p=Q)
    assert np.array_equal(host(Qaux), Qaux_ref)
    Ut = mvk.batch_project(QtT, n, dev(ei), dev(ev), p=Q)
    assert np.array_equal(host(Ut), oracle.batch_project(Qs, ei, ev, p=Q))
    bad = Y.copy()
    bad[B - 1, m // 3] = (int(bad[B - 1, m // 3]) + 5) % Q
    for resp, want in ((Y, [1] * B), (bad, [1] * (B - 1) + [0])):
        outs = [torch.empty((2, s), dtype=torch.int32, device="cuda") for s in (B, B, 2, 2)]
        acc, vL, vR, sL, sR = mvk.batch_verify(dcy, dc2, Qaux, dev(X), dev(resp), dev(ei), dev(ev), Ut, dev(e2i),
                                               dev(e2v), vL=outs[0], vR=outs[1], sL=outs[2], sR=outs[3])
        ref = oracle.batch_verify(cy, c2, Qaux_ref, X, resp, ei, ev, host(Ut), e2i, e2v, p=Q)
        for got, w in zip((vL, vR, sL, sR), ref[2:]):
            assert np.array_equal(host(got), w)
        assert host(acc).tolist() == ref[0].astype(np.uint32).tolist() == want


# ---------------------------------------------------------------------------
# The Sec. 7.1 workload at n = 2^14 (r = 8, t_x = 154): X^, Y^ and Y in full
# (the oracle's product threaded over row blocks), P^T and Q on sampled
# columns (a full oracle keygen would hold 2^31 words of each)
# ---------------------------------------------------------------------------
def test_paper_eval_n16384():
    cfg = synth.PAPER_EVAL
    n = 16384
    _say(f"babybear paper workload n={n} r={cfg['r']} tx={cfg['tx'][n]}")
    inst = Instance(cfg["cid"], n, n, 1, cfg["r"], cfg["tx"][n], cfg["ty"], cfg["ell"], p=Q).to_device()
    mvk.keygen(inst.key, inst.dW)
    g = synth.rng(synth.seed_for(cfg["cid"], 99))
    rows = np.unique(np.concatenate([[0, n - 1], g.integers(0, n, 40)]))
    for i in rows:
        want = oracle.encT(inst.cx, (inst.W[i].astype(np.int64) % Q).astype(np.uint32), p=Q)
        assert np.array_equal(host(inst.key.PT[:, int(i)]), want)
        want = oracle.encT(inst.cy, (inst.W[:, i].astype(np.int64) % Q).astype(np.uint32), p=Q)
        assert np.array_equal(host(inst.key.Q[:, int(i)]), want)
    dXh = mvk.encode(inst.key, inst.dX, inst.dexi, inst.dexv)
    Xh = oracle.encode(inst.cx, inst.X, inst.exi, inst.exv, p=Q)
    assert np.array_equal(host(dXh), Xh)
    T = oracle.threads()
    dYh = mvk.server_eval(inst.dW, dXh, p=Q)
    assert np.array_equal(host(dYh), oracle.server_eval(inst.W, Xh, p=Q, nthreads=T))
    Y, acc, _, _ = mvk.decode_verify(inst.key, dXh, dYh, inst.dexi, inst.dexv, inst.deyi, inst.deyv)
    assert host(acc).tolist() == [1]
    # completeness (Thm. 6.1): the decryption of an honest response is W x
    assert np.array_equal(host(Y), oracle.server_eval(inst.W, inst.X, p=Q, nthreads=T))
    bad = dYh.clone()
    bad[0, int(rows[1])] = (int(bad[0, int(rows[1])]) + 777) % Q
    _, acc2, _, _ = mvk.decode_verify(inst.key, dXh, bad, inst.dexi, inst.dexv, inst.deyi, inst.deyv)
    assert host(acc2).tolist() == [0]
