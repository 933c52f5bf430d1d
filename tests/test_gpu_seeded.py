"""GPU parity of the seeded calls (the library draws the codes, the noise and
the challenges; Protocol pvMVMD, Sec. 6.1; App. B; Sec. 3).

The oracle draws the same randomness from the same seeds with its own
implementation of the sampling specification, then computes Preprocess,
Encrypt, the server product, Verify and Decrypt; every output of the library
is compared with it bit for bit: the code arrays, P^T, Q, the noise, X^, Y,
v_L, v_R and the accept bits (honest and tampered responses), over both fields.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import dev, host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_10264_amd as mvk
    mvk._lib.load()
    mvk._lib.load(mvk.P_BABYBEAR)


def _say(*a):
    print(*a, flush=True)


import paper_2609_10264_amd as mvk  # noqa: E402

CASES = [
    # (m, n, B, r_x, r_y, t_x, t_y, ell, p)
    (256, 256, 1, 2, 2, 8, 31, 2, synth.P),
    (300, 170, 5, 3, 2, 24, 31, 2, synth.P),
    (4096, 4096, 1, 3, 3, 64, 31, 2, synth.P),
    (1000, 900, 16, 3, 3, 64, 31, 3, synth.P),
    (257, 300, 3, 8, 8, 160, 31, 2, synth.P_BABYBEAR),
    (2048, 2048, 1, 8, 8, 159, 31, 2, synth.P_BABYBEAR),
]


@pytest.mark.parametrize("m,n,B,rx,ry,tx,ty,ell,p", CASES)
def test_seeded_path_matches_oracle(m, n, B, rx, ry, tx, ty, ell, p):
    _say(f"seeded m={m} n={n} B={B} r=({rx},{ry}) t=({tx},{ty}) ell={ell} p={p}")
    code_seed, noise_seed, chal_seed = 1000 * m + n, 7 * m + 3, 2**63 + 11 * n
    W = synth.weights(5 * m + n, m, n)
    X = synth.field_uniform(3 * m + n, (B, n), p=p)
    pp = mvk.keygen_seeded(dev(W), rx, ry, code_seed, p=p)
    key = pp.key
    cx = oracle.sample_code(n, rx, code_seed, oracle.TAG_CODE_X, p=p)
    cy = oracle.sample_code(m, ry, code_seed, oracle.TAG_CODE_Y, p=p)
    for c, d in ((cx, key.cx), (cy, key.cy)):
        for name in ("pi1", "pi2", "v1", "v2"):
            assert np.array_equal(host(getattr(d, name)), c[name]), name
    PT, Q = oracle.keygen(W, cx, cy, p=p, nthreads=oracle.threads())
    assert np.array_equal(host(key.PT), PT) and np.array_equal(host(key.Q), Q)

    dXh, st = mvk.encode_seeded(key, dev(X), tx, noise_seed)
    exi, exv = oracle.sample_sparse(B, cx["N"], tx, noise_seed, oracle.TAG_NOISE, p=p)
    torch.cuda.synchronize()
    assert np.array_equal(host(st.idx), exi) and np.array_equal(host(st.val), exv)
    Xh = oracle.encode(cx, X, exi, exv, p=p)
    assert np.array_equal(host(dXh), Xh)

    dYh = mvk.server_eval(mvk.pack_weights(dev(W)), dXh, p=p)
    Yh = oracle.server_eval(W, Xh, p=p, nthreads=oracle.threads())
    assert np.array_equal(host(dYh), Yh)
    eyi, eyv = oracle.sample_sparse(ell, cy["N"], ty, chal_seed, oracle.TAG_CHALLENGE, p=p)
    vL = torch.empty((ell, B), dtype=torch.int32, device="cuda")
    vR = torch.empty_like(vL)
    Y, acc, _, _ = mvk.decode_verify_seeded(key, st, dXh, dYh, ty, ell, chal_seed, vL=vL, vR=vR)
    oacc, ovL, ovR = oracle.verify(cy, Q, Xh, Yh, eyi, eyv, p=p)
    assert np.array_equal(host(vL), ovL) and np.array_equal(host(vR), ovR)
    assert host(acc).tolist() == oacc.astype(np.uint32).tolist() == [1] * B
    Yo = oracle.decode(PT, Yh, exi, exv, p=p)
    assert np.array_equal(host(Y), Yo) and np.array_equal(Yo, oracle.server_eval(W, X, p=p))

    # a tampered response: the oracle's verdict and values, bit for bit
    bad = Yh.copy()
    b = B - 1
    bad[b, m // 3] = (int(bad[b, m // 3]) + 424242) % p
    Y2, acc2, _, _ = mvk.decode_verify_seeded(key, st, dXh, dev(bad), ty, ell, chal_seed, vL=vL, vR=vR)
    oacc2, ovL2, ovR2 = oracle.verify(cy, Q, Xh, bad, eyi, eyv, p=p)
    assert host(acc2).tolist() == oacc2.astype(np.uint32).tolist()
    assert oacc2.tolist() == [True] * (B - 1) + [False]
    assert np.array_equal(host(vL), ovL2) and np.array_equal(host(vR), ovR2)
    assert np.array_equal(host(Y2), oracle.decode(PT, bad, exi, exv, p=p))
    del st, pp


def test_fresh_seeds_draw_new_noise_and_still_decrypt():
    """MVK_SEED_FRESH: each Encrypt gets a seed from the operating system; two
    calls on the same query give different masked queries, both decrypt to W x
    and are accepted under fresh challenges."""
    m, n, B = 512, 384, 2
    W = synth.weights(31, m, n)
    X = synth.field_uniform(32, (B, n))
    pp = mvk.keygen_seeded(dev(W), 3, 3, mvk.SEED_FRESH)
    dW = dev(W)
    outs = []
    for _ in range(2):
        dXh, st = mvk.encode_seeded(pp.key, dev(X), 40, mvk.SEED_FRESH)
        dYh = mvk.server_eval(dW, dXh)
        Y, acc, _, _ = mvk.decode_verify_seeded(pp.key, st, dXh, dYh, 31, 2, mvk.SEED_FRESH)
        torch.cuda.synchronize()
        assert host(acc).tolist() == [1] * B
        assert np.array_equal(host(Y), oracle.server_eval(W, X))
        outs.append((host(dXh), host(st.idx)))
    assert not np.array_equal(outs[0][0], outs[1][0]) and not np.array_equal(outs[0][1], outs[1][1])


def test_seeded_key_works_with_every_call():
    """The key view of a seeded pp is an ordinary key: the prepared path and
    the one-call path with the state's noise give the seeded path's outputs."""
    m, n, B, ty, ell, seed = 640, 512, 4, 31, 2, 99
    W = synth.weights(41, m, n)
    X = synth.field_uniform(42, (B, n))
    pp = mvk.keygen_seeded(dev(W), 3, 3, 5)
    key = pp.key
    dXh, st = mvk.encode_seeded(key, dev(X), 64, 6)
    dYh = mvk.server_eval(dev(W), dXh)
    Y1, acc1, _, _ = mvk.decode_verify_seeded(key, st, dXh, dYh, ty, ell, seed)
    eyi, eyv = oracle.sample_sparse(ell, key.cy.N, ty, seed, oracle.TAG_CHALLENGE)
    Y2, acc2, _, _ = mvk.decode_verify(key, dXh, dYh, st.idx, st.val, dev(eyi), dev(eyv))
    prep = mvk.client_prepare(key, st.idx, st.val, dev(eyi), dev(eyv))
    Xh3 = mvk.encode_masked(key, dev(X), prep)
    Y3, acc3, _, _ = mvk.decode_verify_masked(key, Xh3, mvk.server_eval(dev(W), Xh3), prep)
    torch.cuda.synchronize()
    assert torch.equal(Xh3, dXh)
    for a, b in ((Y1, Y2), (Y1, Y3), (acc1, acc2), (acc1, acc3)):
        assert torch.equal(a, b)
    assert host(acc1).tolist() == [1] * B
