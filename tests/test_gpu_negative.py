"""Soundness on the GPU (Protocol pvMVMD, Thm. 6.1; Lemma 5.1): responses that
are not W x^ for the client's own masked query are rejected, on the one-call,
prepared and seeded paths, and the GPU's v_L, v_R and accept bits equal the
oracle's for each of them.

Dishonest servers: two columns of the response swapped; a column answered
with the response to an earlier query (replay); the product computed with
another matrix of the same shape (a foreign key's W); the right matrix applied
to another query.  Wrong client keys: verifying against the Q of another
matrix, and against a verification code the responses were not keyed with.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import Instance, code, dev, host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_10264_amd as mvk
    mvk._lib.load()
    mvk._lib.load(mvk.P_BABYBEAR)


import paper_2609_10264_amd as mvk  # noqa: E402


def _check(inst, key, Q_orc, Xh, bad, want, tag):
    """One-call and prepared paths on response `bad` against the oracle's
    verdict, which must be `want`."""
    p = inst.p
    ell, B = inst.eyi.shape[0], inst.B
    oacc, ovL, ovR = oracle.verify(inst.cy, Q_orc, Xh, bad, inst.eyi, inst.eyv, p=p)
    assert oacc.tolist() == want, (tag, "oracle")
    vL = torch.empty((ell, B), dtype=torch.int32, device="cuda")
    vR = torch.empty_like(vL)
    dXh, dbad = dev(Xh), dev(bad)
    _, acc, _, _ = mvk.decode_verify(key, dXh, dbad, inst.dexi, inst.dexv, inst.deyi, inst.deyv, vL=vL, vR=vR)
    assert host(acc).tolist() == [int(a) for a in want], (tag, "one-call")
    assert np.array_equal(host(vL), ovL) and np.array_equal(host(vR), ovR), (tag, "one-call v")
    prep = mvk.client_prepare(key, inst.dexi, inst.dexv, inst.deyi, inst.deyv)
    _, acc2, _, _ = mvk.decode_verify_masked(key, dXh, dbad, prep, vL=vL, vR=vR)
    assert host(acc2).tolist() == [int(a) for a in want], (tag, "prepared")
    assert np.array_equal(host(vL), ovL) and np.array_equal(host(vR), ovR), (tag, "prepared v")


@pytest.mark.parametrize("p", [synth.P, synth.P_BABYBEAR], ids=["m31", "babybear"])
def test_dishonest_responses_rejected(p):
    m, n, B = 1000, 900, 6
    inst = Instance(41, m, n, B, 3, 64, 31, 2, p=p).to_device()
    mvk.keygen(inst.key, inst.dW)
    _, Q = oracle.keygen(inst.W, inst.cx, inst.cy, want_P=False, p=p)
    Xh = oracle.encode(inst.cx, inst.X, inst.exi, inst.exv, p=p)
    Yh = oracle.server_eval(inst.W, Xh, p=p)
    assert np.array_equal(host(mvk.server_eval(inst.dW, dev(Xh), p=p)), Yh)
    _check(inst, inst.key, Q, Xh, Yh, [True] * B, "honest")

    swapped = Yh.copy()
    swapped[[1, 4]] = Yh[[4, 1]]
    _check(inst, inst.key, Q, Xh, swapped, [True, False, True, True, False, True], "swapped columns")

    # replay: column 2 answered with the response to an earlier query of the same client
    X_old = synth.field_uniform(4242, (1, n), p=p)
    old = oracle.server_eval(inst.W, oracle.encode(inst.cx, X_old, inst.exi[2:3], inst.exv[2:3], p=p), p=p)
    replay = Yh.copy()
    replay[2] = old[0]
    _check(inst, inst.key, Q, Xh, replay, [True, True, False, True, True, True], "replayed column")

    # the product with another matrix of the same shape (every column wrong)
    W2 = synth.weights(4343, m, n)
    foreign = oracle.server_eval(W2, Xh, p=p)
    _check(inst, inst.key, Q, Xh, foreign, [False] * B, "foreign matrix")

    # the right matrix applied to another query in column 5
    other = Yh.copy()
    other[5] = oracle.server_eval(inst.W, synth.field_uniform(4444, (1, n), p=p), p=p)[0]
    _check(inst, inst.key, Q, Xh, other, [True] * 5 + [False], "another query")


def test_wrong_keys_reject_honest_responses():
    """Honest responses for W checked with the Q of another matrix, and with a
    key whose verification code differs from the one the responses' Q used."""
    m, n, B = 700, 520, 4
    inst = Instance(43, m, n, B, 3, 40, 31, 2).to_device()
    Xh = oracle.encode(inst.cx, inst.X, inst.exi, inst.exv)
    Yh = oracle.server_eval(inst.W, Xh)
    # Q of a foreign matrix under the same codes
    W2 = synth.weights(4545, m, n)
    key2 = mvk.Key.allocate(m, n, code(inst.cx), code(inst.cy))
    mvk.keygen(key2, dev(W2))
    _, Q2 = oracle.keygen(W2, inst.cx, inst.cy, want_P=False)
    _check(inst, key2, Q2, Xh, Yh, [False] * B, "foreign key")
    # a key of W under another verification code: the client's challenges are
    # positions of that code's codewords, so the check compares unrelated values
    cy3 = synth.raa_code(4646, m, 3)
    key3 = mvk.Key.allocate(m, n, code(inst.cx), code(cy3))
    mvk.keygen(key3, inst.dW)
    _, Q3 = oracle.keygen(inst.W, inst.cx, cy3, want_P=False)
    inst3 = Instance(43, m, n, B, 3, 40, 31, 2)
    inst3.cy = cy3
    inst3.to_device()
    # Q3 is consistent with cy3: honest responses pass under (key3, cy3) ...
    _check(inst3, key3, Q3, Xh, Yh, [True] * B, "own code")
    # ... and fail when the client's Q comes from one code and Gy from the other
    mixed = mvk.Key(m, n, key3.cx, inst.key.cy, key3.PT, key3.Q)
    inst4 = Instance(43, m, n, B, 3, 40, 31, 2).to_device()
    _check(inst4, mixed, Q3, Xh, Yh, [False] * B, "mixed codes")


def test_seeded_path_rejects_a_stale_response():
    """Seeded Encrypt twice with fresh noise: the response to the first masked
    query does not pass as the response to the second."""
    m, n, B = 512, 640, 3
    W = synth.weights(4747, m, n)
    X = synth.field_uniform(4848, (B, n))
    pp = mvk.keygen_seeded(dev(W), 3, 3, 77)
    dW = dev(W)
    Xh1, st1 = mvk.encode_seeded(pp.key, dev(X), 48, 1001)
    Xh2, st2 = mvk.encode_seeded(pp.key, dev(X), 48, 1002)
    Yh1 = mvk.server_eval(dW, Xh1)
    _, acc, _, _ = mvk.decode_verify_seeded(pp.key, st2, Xh2, Yh1, 31, 2, 9)
    _, acc_ok, _, _ = mvk.decode_verify_seeded(pp.key, st2, Xh2, mvk.server_eval(dW, Xh2), 31, 2, 9)
    torch.cuda.synchronize()
    assert host(acc).tolist() == [0] * B and host(acc_ok).tolist() == [1] * B
