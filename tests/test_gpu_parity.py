"""GPU parity: every call of the C ABI against the CPU oracle, bit-exact.

All arithmetic is integer mod p, so every comparison is exact equality.
Sizes span several workgroup tiles with ragged tails; the 4096 x 4096 layer
is compared whole here, the larger LLM-layer shapes in test_gpu_fullsize.py.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import Instance, code, dev, host

pytestmark = pytest.mark.gpu
P = synth.P


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_10264_amd as mvk  # noqa: F401  (raises if libmvk.so is missing)
    mvk._lib.load()


def _say(*a):
    print(*a, flush=True)


import paper_2609_10264_amd as mvk  # noqa: E402


# ---------------------------------------------------------------------------
# server_eval
# ---------------------------------------------------------------------------
SERVER_SHAPES = [
    (1, 1, 1), (3, 5, 1), (17, 33, 2), (256, 256, 1), (257, 4099, 1), (64, 4096, 3), (16, 8192, 1),
    (100, 160, 5), (300, 1000, 16), (31, 2048, 64), (4096, 4096, 1), (33, 12345, 4), (50, 4112, 7),
    (129, 300, 17), (70, 999, 65), (16, 128, 130), (200, 4096, 32), (1000, 8192, 64),
    # 5..16 queries with the digit tiles kept in LDS: split k-ranges, ragged
    # rows, and a row length whose k-ranges no longer fit (other kernel)
    (257, 11008, 8), (300, 4096, 12), (64, 16448, 8), (129, 8192, 16),
]


PATHS = ["auto", "valu", "mfma"]


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("m,n,B", SERVER_SHAPES)
def test_server_eval_matches_oracle(m, n, B, path):
    _say(f"server_eval m={m} n={n} B={B} path={path}")
    W = synth.weights(11 * m + n, m, n, lo=-128, hi=127)
    X = synth.field_uniform(13 * n + B, (B, n))
    got = host(mvk.server_eval(dev(W), dev(X), path=path))
    assert np.array_equal(got, oracle.server_eval(W, X))


def _pack_host(W):
    """The packed server layout written out with numpy (tiles of 16 rows x 64
    columns, lane l = 16*(column quarter) + row within the tile, zero padded)."""
    m, n = W.shape
    nrt, nkb = -(-m // 16), -(-n // 64)
    pad = np.zeros((nrt * 16, nkb * 64), dtype=np.int8)
    pad[:m, :n] = W
    t = pad.reshape(nrt, 16, nkb, 4, 16).transpose(0, 2, 3, 1, 4)
    return t.reshape(-1)


@pytest.mark.parametrize("m,n", [(1, 1), (17, 100), (64, 4096), (33, 12345)])
def test_pack_weights_layout(m, n):
    W = synth.weights(400 + m, m, n)
    pw = mvk.pack_weights(dev(W))
    want = _pack_host(W)
    got = pw.data.cpu().numpy()[: want.size]
    assert got.size == want.size == mvk._lib.load().mvk_packed_weight_bytes(m, n)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("m,n,B", SERVER_SHAPES)
def test_server_eval_packed_matches_oracle(m, n, B):
    _say(f"server_eval packed m={m} n={n} B={B}")
    W = synth.weights(100 + m + n, m, n)
    X = synth.field_uniform(200 + B + n, (B, n))
    got = host(mvk.server_eval(mvk.pack_weights(dev(W)), dev(X)))
    assert np.array_equal(got, oracle.server_eval(W, X))


# 17..32 queries on packed W with at least 192 blocks of 128 rows: the
# 32x32x32 wide-tile kernel (no k split).  Ragged rows (24600, 25000, 24704)
# and columns (1000 and 520: not multiples of 64, 1000 not of 16), 32, 20 and
# 17 queries; 8192 columns.  Next to them 33..64 queries on the streamed
# kernel: 64 and 33 queries of those shapes, 200 columns (four k-blocks, the
# last one ragged), 40960 rows, 57 queries at 20736 x 4096.
WIDE_SHAPES = [(24576, 1000, 32), (24600, 640, 25), (25000, 520, 20), (24576, 8192, 32), (24704, 64, 17),
               (24576, 1000, 64), (24600, 640, 33), (20480, 200, 64), (40960, 256, 40), (20736, 4096, 57)]


@pytest.mark.parametrize("m,n,B", WIDE_SHAPES)
def test_server_eval_wide_tiles_match_oracle(m, n, B):
    _say(f"server_eval wide tiles m={m} n={n} B={B}")
    W = synth.weights(300 + m + n, m, n)
    X = synth.field_uniform(301 + B + n, (B, n))
    got = host(mvk.server_eval(mvk.pack_weights(dev(W)), dev(X)))
    assert np.array_equal(got, oracle.server_eval(W, X, nthreads=oracle.threads()))


def test_server_eval_group_wide_tiles_match_oracle():
    """A row stack of two matrices (12800 rows each) with 30 queries: the
    wide-tile kernel writes each matrix's rows to its own output."""
    mg, n, B = 12800, 700, 30
    Ws = [synth.weights(310 + g, mg, n) for g in range(2)]
    X = synth.field_uniform(312, (B, n))
    outs = mvk.server_eval_group(mvk.pack_weights_group([dev(W) for W in Ws]), 2, dev(X))
    for W, Y in zip(Ws, outs):
        assert np.array_equal(host(Y), oracle.server_eval(W, X, nthreads=oracle.threads()))


def test_server_eval_group_64_queries_match_oracle():
    """A row stack of two matrices of 12304 rows (a row block of the streamed
    kernel straddles them) with 50 queries: each matrix's rows go to its own
    output."""
    mg, n, B = 12304, 700, 50
    Ws = [synth.weights(320 + g, mg, n) for g in range(2)]
    X = synth.field_uniform(322, (B, n))
    outs = mvk.server_eval_group(mvk.pack_weights_group([dev(W) for W in Ws]), 2, dev(X))
    for W, Y in zip(Ws, outs):
        assert np.array_equal(host(Y), oracle.server_eval(W, X, nthreads=oracle.threads()))


def test_server_eval_16384_single_query_matches_oracle():
    """The single-query shape the bench measures against the read floor
    (16384 x 16384, packed W, one column): Y^ in full against the oracle,
    threaded over row blocks."""
    m = n = 16384
    _say(f"server_eval {m}x{n} B=1 packed")
    W = synth.weights(330, m, n)
    X = synth.field_uniform(331, (1, n))
    got = host(mvk.server_eval(mvk.pack_weights(dev(W)), dev(X)))
    assert np.array_equal(got, oracle.server_eval(W, X, nthreads=oracle.threads()))


@pytest.mark.parametrize("m,n,B", [(4096, 16384, 8), (4096, 16384, 16), (24576, 1024, 32), (20480, 2048, 64)])
@pytest.mark.parametrize("wv", [-128, 127])
def test_server_eval_batched_extremes_closed_form(m, n, B, wv):
    """Constant W = wv (packed) against B queries, each a constant at an
    extreme of the balanced digits (every digit -128 or 127, the centring
    boundary, 0, 1, p - 1): every row of query q is n wv x_q mod p, on the
    digits-stationary kernel (8 and 16 queries), the wide-tile kernel (32) and
    the streamed kernel (64)."""
    xs = [P - 8421504, 8421504 - 1, P - 1, 1, 0, 1073741823, 1073741824, 2139062143]
    xs = [xs[q % len(xs)] if q < len(xs) else (xs[q % len(xs)] + q * 7919) % P for q in range(B)]
    _say(f"server_eval batched extremes m={m} n={n} B={B} w={wv}")
    W = torch.full((m, n), wv, dtype=torch.int8, device="cuda")
    X = torch.tensor(np.repeat(np.array(xs, dtype=np.uint32)[:, None], n, axis=1).view(np.int32), device="cuda")
    got = host(mvk.server_eval(mvk.pack_weights(W), X))
    want = np.array([(n * wv * x) % P for x in xs], dtype=np.uint32)
    assert np.array_equal(got, np.repeat(want[:, None], m, axis=1))


@pytest.mark.parametrize("B", [5, 16, 20, 64])
@pytest.mark.parametrize("wv", [-128, 127])
def test_server_eval_batched_extremes_at_max_n(B, wv):
    """n at the exactness limit (every digit-plane sum up to n 128 128 - 1 <
    2^31) on the batched kernels: 300 rows of constant W = wv, packed, against
    B queries, each a constant at an extreme of the balanced digits; every
    row of query q is n wv x_q mod p.  At this n no k-range of digit tiles
    fits in LDS, so every B takes the streamed kernel (2, 4, 8 and 16 digit
    tiles), k split where its plan splits it."""
    m, n = 300, mvk.MVK_MAX_N
    base = [P - 8421504, 1073741823, 1073741824, P - 1, 1, 0, 8421503, 2139062143]
    xs = [base[q % len(base)] for q in range(B)]
    _say(f"server_eval batched extremes n={n} B={B} w={wv}")
    W = torch.full((m, n), wv, dtype=torch.int8, device="cuda")
    X = torch.tensor(np.repeat(np.array(xs, dtype=np.uint32)[:, None], n, axis=1).view(np.int32), device="cuda")
    got = host(mvk.server_eval(mvk.pack_weights(W), X))
    want = np.array([(n * wv * x) % P for x in xs], dtype=np.uint32)
    assert np.array_equal(got, np.repeat(want[:, None], m, axis=1))


@pytest.mark.parametrize("path", ["valu", "mfma"])
@pytest.mark.parametrize("wv,xv", [(-128, P - 8421504), (127, P - 1), (-127, P - 1), (-128, 1073741823),
                                   (127, 1073741824), (-1, 0)])
def test_server_eval_extremes(wv, xv, path):
    # n at the exactness limit: every digit-plane sum reaches n * 128 * 128 - 1 < 2^31
    m, n = 5, mvk.MVK_MAX_N
    _say(f"server_eval extreme w={wv} x={xv} n={n} path={path}")
    W = np.full((m, n), wv, dtype=np.int8)
    X = np.full((2, n), xv, dtype=np.uint32)
    X[1, ::3] = 0
    got = host(mvk.server_eval(dev(W), dev(X), path=path))
    assert np.array_equal(got, oracle.server_eval(W, X))


def test_server_eval_empty_and_limits():
    W = dev(synth.weights(1, 8, 0))
    X = torch.zeros((2, 0), dtype=torch.int32, device="cuda")
    Y = mvk.server_eval(W, X, out=torch.full((2, 8), 7, dtype=torch.int32, device="cuda"))
    assert not Y.any()  # empty sum
    Y0 = torch.full((0, 8), 7, dtype=torch.int32, device="cuda")
    mvk.server_eval(dev(synth.weights(1, 8, 4)), torch.zeros((0, 4), dtype=torch.int32, device="cuda"), out=Y0)
    with pytest.raises(mvk.MvkError):
        mvk.server_eval(torch.zeros((2, mvk.MVK_MAX_N + 1), dtype=torch.int8, device="cuda"),
                        torch.zeros((1, mvk.MVK_MAX_N + 1), dtype=torch.int32, device="cuda"))


def test_server_eval_closed_forms():
    n = 1000
    X = synth.field_uniform(5, (3, n))
    I = np.eye(n, dtype=np.int8)
    assert np.array_equal(host(mvk.server_eval(dev(I), dev(X))), X)
    M = np.full((7, n), -1, dtype=np.int8)
    want = np.array([[(-sum(int(v) for v in x)) % P] * 7 for x in X], dtype=np.uint32)
    assert np.array_equal(host(mvk.server_eval(dev(M), dev(X))), want)


def test_server_eval_repeatable_and_noncontiguous_offsets():
    # outputs written at an offset inside a larger buffer; repeated runs are bitwise equal
    m, n, B = 130, 520, 3
    W = synth.weights(21, m, n)
    X = synth.field_uniform(22, (B, n))
    big = torch.zeros((B * m + 64,), dtype=torch.int32, device="cuda")
    out = big[64:].view(B, m)
    a = host(mvk.server_eval(dev(W), dev(X), out=out))
    b = host(mvk.server_eval(dev(W), dev(X)))
    assert np.array_equal(a, b) and np.array_equal(a, oracle.server_eval(W, X))
    assert not big[:64].any()


@pytest.mark.parametrize("nbytes", [16, 4096, 16 * 262144 * 8 + 48, 16777216 + 1024])
def test_stream_read_checksum(nbytes):
    """The calibration read covers every byte once: the XOR of its sink words is
    the XOR of the buffer's 32-bit words (ragged passes included)."""
    data = synth.weights(nbytes, 1, nbytes)
    sink = mvk.stream_read(dev(data))
    want = np.bitwise_xor.reduce(data.view(np.uint32).ravel())
    assert int(np.bitwise_xor.reduce(host(sink))) == int(want)


def test_validate_mode_rejects_noncanonical_inputs():
    """MVK_VALIDATE=1: a field input >= p is an error (MVK_ERANGE) before any
    work; canonical inputs give the usual results."""
    inst = Instance(61, 200, 300, 2, 2, 5).to_device()
    mvk.keygen(inst.key, inst.dW)
    Xh = mvk.encode(inst.key, inst.dX, inst.dexi, inst.dexv)
    Yh = mvk.server_eval(inst.dW, Xh)
    torch.cuda.synchronize()
    os.environ["MVK_VALIDATE"] = "1"
    try:
        assert np.array_equal(host(mvk.server_eval(inst.dW, Xh)), host(Yh))
        bad = Xh.clone()
        bad[1, 7] = P
        for call in (lambda: mvk.server_eval(inst.dW, bad),
                     lambda: mvk.encode(inst.key, bad, inst.dexi, inst.dexv),
                     lambda: mvk.decode_verify(inst.key, bad, Yh, inst.dexi, inst.dexv, inst.deyi, inst.deyv)):
            with pytest.raises(mvk.MvkError) as err:
                call()
            assert err.value.status == mvk._lib.MVK_ERANGE
        badY = Yh.clone()
        badY[0, 3] = -1  # 0xffffffff
        with pytest.raises(mvk.MvkError):
            mvk.decode_verify(inst.key, Xh, badY, inst.dexi, inst.dexv, inst.deyi, inst.deyv)
        Y, acc, _, _ = mvk.decode_verify(inst.key, Xh, Yh, inst.dexi, inst.dexv, inst.deyi, inst.deyv)
        assert host(acc).tolist() == [1, 1]
    finally:
        del os.environ["MVK_VALIDATE"]


# ---------------------------------------------------------------------------
# RAA encoding / syndrome
# ---------------------------------------------------------------------------
# N = k*r spans every single-workgroup tile size (N <= 4096, 8192, 12288,
# 16384, each with a ragged last row) and the segmented path above 16384.
@pytest.mark.parametrize("k,r,count", [(1, 1, 1), (5, 2, 3), (256, 2, 2), (1000, 3, 4), (4097, 4, 2), (700, 5, 65),
                                         (6000, 4, 2), (5056, 4, 1), (2048, 4, 2), (2731, 3, 2), (4096, 3, 3),
                                         (5461, 3, 1), (4096, 4, 2), (16384, 1, 1), (1366, 6, 2)])
def test_raa_encode_and_syndrome(k, r, count):
    _say(f"raa k={k} r={r} count={count}")
    c = synth.raa_code(300 + k + r, k, r)
    w = synth.field_uniform(301 + k, (count, k))
    v = synth.field_uniform(302 + k, (count, k * r))
    dc = code(c)
    got_e = host(mvk.raa_encode(dc, dev(w)))
    got_s = host(mvk.raa_syndrome(dc, dev(v)))
    for i in range(count):
        assert np.array_equal(got_e[i], oracle.encT(c, w[i]))
        assert np.array_equal(got_s[i], oracle.syn(c, v[i]))


def test_raa_identity_closed_form():
    N = 5000
    c = synth.identity_code(N, 1)
    e0 = np.zeros((1, N), dtype=np.uint32)
    e0[0, 0] = 1
    assert host(mvk.raa_encode(code(c), dev(e0)))[0].tolist() == list(range(1, N + 1))
    assert host(mvk.raa_syndrome(code(c), dev(e0[:, ::-1].copy())))[0].tolist() == [N - i for i in range(N)]


# ---------------------------------------------------------------------------
# keygen / encode / decode_verify on small and ragged shapes
# ---------------------------------------------------------------------------
SMALL = [  # cid, m, n, B, r, tx
    (0, 256, 256, 1, 2, 8),
    (50, 257, 130, 3, 3, 5),
    (51, 64, 1000, 2, 4, 17),
    (52, 1000, 64, 5, 1, 3),
]


@pytest.mark.parametrize("cid,m,n,B,r,tx", SMALL)
def test_protocol_small(cid, m, n, B, r, tx):
    _say(f"protocol cid={cid} m={m} n={n} B={B} r={r} tx={tx}")
    inst = Instance(cid, m, n, B, r, tx).to_device()
    mvk.keygen(inst.key, inst.dW)
    PT, Q = oracle.keygen(inst.W, inst.cx, inst.cy)
    assert np.array_equal(host(inst.key.PT), PT)
    assert np.array_equal(host(inst.key.Q), Q)
    dXh = mvk.encode(inst.key, inst.dX, inst.dexi, inst.dexv)
    Xh = oracle.encode(inst.cx, inst.X, inst.exi, inst.exv)
    assert np.array_equal(host(dXh), Xh)
    dYh = mvk.server_eval(inst.dW, dXh)
    Yh = oracle.server_eval(inst.W, Xh)
    assert np.array_equal(host(dYh), Yh)
    ell = inst.eyi.shape[0]
    vL = torch.empty((ell, B), dtype=torch.int32, device="cuda")
    vR = torch.empty_like(vL)
    Y, acc, vL, vR = mvk.decode_verify(inst.key, dXh, dYh, inst.dexi, inst.dexv, inst.deyi, inst.deyv, vL=vL, vR=vR)
    oacc, ovL, ovR = oracle.verify(inst.cy, Q, Xh, Yh, inst.eyi, inst.eyv)
    assert np.array_equal(host(vL), ovL) and np.array_equal(host(vR), ovR)
    assert host(acc).tolist() == oacc.astype(np.uint32).tolist() == [1] * B
    assert np.array_equal(host(Y), oracle.decode(PT, Yh, inst.exi, inst.exv))
    assert np.array_equal(host(Y), oracle.server_eval(inst.W, inst.X))

    # tampered responses: one changed coordinate per column in turn
    pos, delta = synth.tamper_delta(synth.seed_for(cid, synth.PURPOSE_TAMPER), B, m)
    for b in range(B):
        bad = Yh.copy()
        bad[b, pos[b]] = (int(bad[b, pos[b]]) + int(delta[b])) % P
        Yb, accb, vLb, vRb = mvk.decode_verify(inst.key, dXh, dev(bad), inst.dexi, inst.dexv, inst.deyi, inst.deyv,
                                               vL=vL, vR=vR)
        oacc, ovL, ovR = oracle.verify(inst.cy, Q, Xh, bad, inst.eyi, inst.eyv)
        assert host(accb).tolist() == oacc.astype(np.uint32).tolist()
        assert not oacc[b]
        assert np.array_equal(host(vLb), ovL) and np.array_equal(host(vRb), ovR)
        assert np.array_equal(host(Yb), oracle.decode(PT, bad, inst.exi, inst.exv))


# Sparse syndromes (encode: one per column; verify_prepare: one per
# repetition) at block lengths in every tile size of the single-workgroup
# kernel and in the segmented range.
@pytest.mark.parametrize("n,r,B,tx", [(1366, 3, 2, 64), (2048, 4, 3, 7), (4096, 3, 1, 64), (5461, 3, 2, 128),
                                       (4096, 4, 1, 100), (4097, 4, 2, 64), (8192, 4, 1, 128), (16384, 1, 1, 1)])
def test_sparse_syndrome_lengths(n, r, B, tx):
    _say(f"sparse syndrome n={n} r={r} B={B} tx={tx}")
    # the same shape as privacy code (n) and as verification code (m = n)
    inst = Instance(70 + r, n, n, B, r, tx, ty=31, ell=3).to_device()
    Xh = mvk.encode(inst.key, inst.dX, inst.dexi, inst.dexv)
    assert np.array_equal(host(Xh), oracle.encode(inst.cx, inst.X, inst.exi, inst.exv))
    R = host(mvk.verify_prepare(inst.key, inst.deyi, inst.deyv))
    for q in range(inst.eyi.shape[0]):
        e = np.zeros(inst.cy["N"], dtype=np.uint32)
        e[inst.eyi[q]] = inst.eyv[q]
        assert np.array_equal(R[q], oracle.syn(inst.cy, e)), q


def test_prepared_verify_matches_unprepared():
    """decode_verify with R from verify_prepare (on another stream) = decode_verify."""
    inst = Instance(53, 700, 333, 4, 3, 9, ell=2).to_device()
    mvk.keygen(inst.key, inst.dW)
    PT, Q = oracle.keygen(inst.W, inst.cx, inst.cy)
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        R = mvk.verify_prepare(inst.key, inst.deyi, inst.deyv, stream=side)
    dXh = mvk.encode(inst.key, inst.dX, inst.dexi, inst.dexv)
    Xh = host(dXh)
    Yh = oracle.server_eval(inst.W, Xh)
    pos, delta = synth.tamper_delta(synth.seed_for(53, synth.PURPOSE_TAMPER), 4, 700)
    Yh[2, pos[2]] = (int(Yh[2, pos[2]]) + int(delta[2])) % P
    torch.cuda.current_stream().wait_stream(side)
    outs = []
    for RR in (None, R):
        vL = torch.empty((2, 4), dtype=torch.int32, device="cuda")
        vR = torch.empty_like(vL)
        Y, acc, vL, vR = mvk.decode_verify(inst.key, dXh, dev(Yh), inst.dexi, inst.dexv, inst.deyi, inst.deyv,
                                           vL=vL, vR=vR, R=RR)
        outs.append([host(t) for t in (Y, acc, vL, vR)])
    oacc, ovL, ovR = oracle.verify(inst.cy, Q, Xh, Yh, inst.eyi, inst.eyv)
    for Y, acc, vL, vR in outs:
        assert acc.tolist() == oacc.astype(np.uint32).tolist() == [1, 1, 0, 1]
        assert np.array_equal(vL, ovL) and np.array_equal(vR, ovR)
        assert np.array_equal(Y, oracle.decode(PT, Yh, inst.exi, inst.exv))


# Decrypt + Verify with the challenge syndromes r_q = Gy e_q computed in the
# same launch: block lengths Ny = ry*m in each tile size of that kernel
# (<= 4096, 8192, 12288, 16384 positions) and past it, and batches whose grid
# does not fit one wave of resident workgroups (both of those take the separate
# syndrome launch).  Two calls in a row, the second with a tampered column,
# check that each launch leaves its completion counters at zero.
@pytest.mark.parametrize("m,ry,B,ell", [(1000, 4, 2, 3), (4096, 2, 1, 2), (2731, 3, 3, 5), (4096, 3, 2, 16),
                                        (4096, 4, 1, 1), (16384, 1, 1, 2), (5462, 3, 1, 2), (4096, 3, 9, 2)])
def test_decode_verify_syndrome_in_launch(m, ry, B, ell):
    _say(f"decode_verify m={m} ry={ry} B={B} ell={ell}")
    inst = Instance(55, m, 64, B, 2, 9, ty=31, ell=ell, ry=ry).to_device()
    mvk.keygen(inst.key, inst.dW)
    PT, Q = oracle.keygen(inst.W, inst.cx, inst.cy)
    dXh = mvk.encode(inst.key, inst.dX, inst.dexi, inst.dexv)
    Xh = host(dXh)
    Yh = oracle.server_eval(inst.W, Xh)
    bad = Yh.copy()
    bad[0, m - 1] = (int(bad[0, m - 1]) + 1) % P
    for resp, want in ((Yh, [1] * B), (bad, [0] + [1] * (B - 1))):
        vL = torch.empty((ell, B), dtype=torch.int32, device="cuda")
        vR = torch.empty_like(vL)
        Y, acc, vL, vR = mvk.decode_verify(inst.key, dXh, dev(resp), inst.dexi, inst.dexv, inst.deyi, inst.deyv,
                                           vL=vL, vR=vR)
        oacc, ovL, ovR = oracle.verify(inst.cy, Q, Xh, resp, inst.eyi, inst.eyv)
        assert oacc.astype(np.uint32).tolist() == want
        assert np.array_equal(host(vL), ovL) and np.array_equal(host(vR), ovR)
        assert host(acc).tolist() == want
        assert np.array_equal(host(Y), oracle.decode(PT, resp, inst.exi, inst.exv))


@pytest.mark.parametrize("m,ry,B,misalign", [(6000, 3, 48, False), (6000, 3, 48, True), (6001, 3, 48, False),
                                             (6000, 3, 3, False), (1000, 4, 64, False), (1000, 4, 64, True),
                                             (998, 4, 64, False)])
def test_decode_widths(m, ry, B, misalign):
    """The decode role with four output columns per lane (m a multiple of 4,
    every row array 16-byte aligned and B * ceil(m/256) >= 256: 16-byte
    gathers, ragged 256-column tail) and with one (m not a multiple of 4, Y 4
    bytes past an alignment, or few columns), in the launch without
    (Ny > 16384) and with the challenge syndromes."""
    _say(f"decode widths m={m} ry={ry} B={B} misalign={misalign}")
    ell = 2
    inst = Instance(57, m, 96, B, 2, 9, ty=31, ell=ell, ry=ry).to_device()
    mvk.keygen(inst.key, inst.dW)
    PT, Q = oracle.keygen(inst.W, inst.cx, inst.cy)
    dXh = mvk.encode(inst.key, inst.dX, inst.dexi, inst.dexv)
    Xh = host(dXh)
    Yh = oracle.server_eval(inst.W, Xh)
    bad = Yh.copy()
    bad[1, m - 1] = (int(bad[1, m - 1]) + 1) % P
    for resp, want in ((Yh, [1] * B), (bad, [1, 0] + [1] * (B - 2))):
        flat = torch.full((B * m + 4,), -1, dtype=torch.int32, device="cuda")
        off = 1 if misalign else 0
        Yout = flat[off: off + B * m].view(B, m)
        Y, acc, _, _ = mvk.decode_verify(inst.key, dXh, dev(resp), inst.dexi, inst.dexv, inst.deyi, inst.deyv,
                                         Y=Yout)
        assert host(acc).tolist() == want
        assert np.array_equal(host(Y), oracle.decode(PT, resp, inst.exi, inst.exv))
        rest = flat.cpu().numpy()
        assert (rest[:off] == -1).all() and (rest[off + B * m:] == -1).all()


@pytest.mark.parametrize("ell,ty", [(1, 31), (3, 5), (5, 31), (16, 2)])
def test_verify_repetition_counts(ell, ty):
    """Work-item split of the verify role for 1..16 repetitions (the maximum)."""
    _say(f"verify ell={ell} ty={ty}")
    inst = Instance(54, 130, 200, 3, 2, 4, ty=ty, ell=ell).to_device()
    mvk.keygen(inst.key, inst.dW)
    _, Q = oracle.keygen(inst.W, inst.cx, inst.cy)
    dXh = mvk.encode(inst.key, inst.dX, inst.dexi, inst.dexv)
    Xh = host(dXh)
    Yh = oracle.server_eval(inst.W, Xh)
    Yh[1, 7] = (int(Yh[1, 7]) + 1) % P
    vL = torch.empty((ell, 3), dtype=torch.int32, device="cuda")
    vR = torch.empty_like(vL)
    _, acc, vL, vR = mvk.decode_verify(inst.key, dXh, dev(Yh), inst.dexi, inst.dexv, inst.deyi, inst.deyv,
                                       vL=vL, vR=vR)
    oacc, ovL, ovR = oracle.verify(inst.cy, Q, Xh, Yh, inst.eyi, inst.eyv)
    assert np.array_equal(host(vL), ovL) and np.array_equal(host(vR), ovR)
    assert host(acc).tolist() == oacc.astype(np.uint32).tolist()


def test_encode_without_noise_is_identity():
    inst = Instance(60, 40, 50, 2, 3, 0).to_device()
    empty = torch.zeros((2, 0), dtype=torch.int32, device="cuda")
    Xh = mvk.encode(inst.key, inst.dX, empty, empty)
    assert np.array_equal(host(Xh), inst.X)


# ---------------------------------------------------------------------------
# LLM-layer shapes at full size
# ---------------------------------------------------------------------------
def test_attn4096_full():
    """4096 x 4096, one query column, r = 3, t_x = 64: whole outputs compared."""
    cfg = synth.CONFIGS["attn4096"]
    _say("attn4096 full compare")
    inst = Instance(cfg["cid"], cfg["m"], cfg["n"], cfg["B"], cfg["r"], cfg["tx"], cfg["ty"], cfg["ell"]).to_device()
    mvk.keygen(inst.key, inst.dW)
    PT, Q = oracle.keygen(inst.W, inst.cx, inst.cy)
    assert np.array_equal(host(inst.key.PT), PT)
    assert np.array_equal(host(inst.key.Q), Q)
    dXh = mvk.encode(inst.key, inst.dX, inst.dexi, inst.dexv)
    Xh = oracle.encode(inst.cx, inst.X, inst.exi, inst.exv)
    assert np.array_equal(host(dXh), Xh)
    dYh = mvk.server_eval(inst.dW, dXh)
    Yh = oracle.server_eval(inst.W, Xh)
    assert np.array_equal(host(dYh), Yh)
    vL = torch.empty((2, 1), dtype=torch.int32, device="cuda")
    vR = torch.empty_like(vL)
    Y, acc, vL, vR = mvk.decode_verify(inst.key, dXh, dYh, inst.dexi, inst.dexv, inst.deyi, inst.deyv, vL=vL, vR=vR)
    oacc, ovL, ovR = oracle.verify(inst.cy, Q, Xh, Yh, inst.eyi, inst.eyv)
    assert np.array_equal(host(vL), ovL) and np.array_equal(host(vR), ovR) and host(acc).tolist() == [1]
    assert np.array_equal(host(Y), oracle.decode(PT, Yh, inst.exi, inst.exv))


# ---------------------------------------------------------------------------
# several matrices sharing their queries in one launch
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("G,m,n,B", [(1, 33, 300, 8), (2, 16, 64, 1), (3, 4096, 4096, 8), (2, 11008, 4096, 8),
                                     (3, 4096, 4096, 1), (4, 256, 1000, 3), (2, 512, 4160, 16), (3, 160, 2048, 40),
                                     (2, 1024, 8192, 64), (4, 48, 130, 70)])
def test_server_eval_group_matches_separate_products(G, m, n, B):
    _say(f"server_eval_group G={G} m={m} n={n} B={B}")
    Ws = [synth.weights(600 + 7 * g + m, m, n, lo=-128, hi=127) for g in range(G)]
    X = synth.field_uniform(700 + n + B, (B, n))
    dX = dev(X)
    stackW = mvk.pack_weights_group([dev(W) for W in Ws])
    outs = mvk.server_eval_group(stackW, G, dX)
    for g, W in enumerate(Ws):
        want = mvk.server_eval(mvk.pack_weights(dev(W)), dX)
        assert torch.equal(outs[g], want), g
    # one of them against the oracle as well
    assert np.array_equal(host(outs[G - 1]), oracle.server_eval(Ws[G - 1], X))
