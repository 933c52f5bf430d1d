"""GPU parity of batch verification (Protocol Batch-vMVMD): preprocessing,
the server's challenge projection and the client checks against the oracle,
bit-exact, with the protocol's rejection cases."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import code, dev, host

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


class Batch:
    """B claims M_b x_b = y_b under one verification code (as the oracle pins build them)."""

    def __init__(self, cid, m, n, B, r, r2, t=31, ell=2, t2=31, ell2=2):
        self.m, self.n, self.B = m, n, B
        sd = lambda purpose, sub=0: synth.seed_for(cid, purpose, sub)  # noqa: E731
        self.Ws = [synth.weights(sd(synth.PURPOSE_W, b), m, n) for b in range(B)]
        self.X = synth.field_uniform(sd(synth.PURPOSE_X), (B, n))
        self.cx = synth.raa_code(sd(synth.PURPOSE_CX), n, 2)
        self.cy = synth.raa_code(sd(synth.PURPOSE_CY), m, r)
        self.c2 = synth.raa_code(sd(synth.PURPOSE_C2), B * n, r2)
        self.Y = np.concatenate([oracle.server_eval(W, self.X[b:b + 1]) for b, W in enumerate(self.Ws)])
        self.ei, self.ev = synth.sparse(sd(synth.PURPOSE_CHAL), ell, self.cy["N"], t)
        self.e2i, self.e2v = synth.sparse(sd(synth.PURPOSE_CHAL2), ell2, self.c2["N"], t2)
        self.Qs = np.stack([oracle.keygen(W, self.cx, self.cy, want_P=False)[1] for W in self.Ws])

    def device(self):
        cx, cy = code(self.cx), code(self.cy)
        keys = []
        for W in self.Ws:
            k = mvk.Key.allocate(self.m, self.n, cx, cy)
            mvk.keygen(k, dev(W))
            keys.append(k)
        self.keys, self.dcy, self.dc2 = keys, cy, code(self.c2)
        return self


SHAPES = [  # cid, m, n, B, r, r2
    (100, 40, 24, 3, 3, 2),
    (101, 1000, 300, 4, 3, 2),
    (102, 6000, 96, 2, 3, 2),     # primary block length 18000: segmented syndromes
    (103, 500, 5000, 2, 2, 2),    # secondary block length 20000: segmented syndromes
    (104, 300, 75, 3, 3, 2),      # B*n = 225: 4-byte gathers of the projection
]


@pytest.mark.parametrize("N,n,B,ell", [(300, 4000, 4, 5), (200, 4096, 4, 5), (300, 1001, 3, 2)])
def test_batch_project_widths(N, n, B, ell):
    """The projection's row gathers with 16-byte loads (B*n a multiple of 4 and
    more than 1024 64-column items: 256 columns per item, ragged at
    B*n = 16000) and with 4-byte loads (few items, or B*n odd)."""
    _say(f"batch project N={N} n={n} B={B} ell={ell}")
    Qs = synth.field_uniform(900 + n, (B, N, n))
    ei, ev = synth.sparse(901 + n, ell, N, 31)
    QtT = dev(np.ascontiguousarray(np.concatenate(list(Qs), axis=1)))
    Ut = mvk.batch_project(QtT, n, dev(ei), dev(ev))
    assert np.array_equal(host(Ut), oracle.batch_project(Qs, ei, ev))


@pytest.mark.parametrize("cid,m,n,B,r,r2", SHAPES)
def test_batch_verification_matches_oracle(cid, m, n, B, r, r2):
    _say(f"batch verify cid={cid} m={m} n={n} B={B} r={r} r2={r2}")
    bt = Batch(cid, m, n, B, r, r2).device()
    QtT, Qaux = mvk.batch_preprocess([k.Q for k in bt.keys], bt.dc2)
    Qaux_ref = oracle.batch_aux(bt.Qs, bt.c2)
    assert np.array_equal(host(QtT), np.concatenate(list(bt.Qs), axis=1))
    assert np.array_equal(host(Qaux), Qaux_ref)
    Ut = mvk.batch_project(QtT, n, dev(bt.ei), dev(bt.ev))
    Ut_ref = oracle.batch_project(bt.Qs, bt.ei, bt.ev)
    assert np.array_equal(host(Ut), Ut_ref)
    ell, ell2 = bt.ei.shape[0], bt.e2i.shape[0]

    def run(Y, Ut_used):
        outs = [torch.empty(s, dtype=torch.int32, device="cuda") for s in ((ell, B), (ell, B), (ell, ell2), (ell, ell2))]
        acc, vL, vR, sL, sR = mvk.batch_verify(bt.dcy, bt.dc2, Qaux, dev(bt.X), dev(Y), dev(bt.ei), dev(bt.ev),
                                               Ut_used, dev(bt.e2i), dev(bt.e2v), vL=outs[0], vR=outs[1],
                                               sL=outs[2], sR=outs[3])
        ref = oracle.batch_verify(bt.cy, bt.c2, Qaux_ref, bt.X, Y, bt.ei, bt.ev, host(Ut_used), bt.e2i, bt.e2v)
        for got, want in zip((vL, vR, sL, sR), ref[2:]):
            assert np.array_equal(host(got), want)
        assert host(acc).tolist() == ref[0].astype(np.uint32).tolist()
        return host(acc).tolist()

    assert run(bt.Y, Ut) == [1] * B
    # a wrong claim: only that claim is rejected
    bad = bt.Y.copy()
    bad[B - 1, m // 3] = (int(bad[B - 1, m // 3]) + 5) % P
    assert run(bad, Ut) == [1] * (B - 1) + [0]
    # a wrong projection: the secondary checks reject the batch
    Ut2 = Ut.clone()
    Ut2[0, 7] = (int(Ut2[0, 7].item()) + 1) % P
    assert run(bt.Y, Ut2) == [0] * B


def test_batch_consistent_forgery_rejected():
    """The server knows the primary challenges: it changes claim 0 and its
    projection so that every original check passes; the secondary checks,
    drawn after, reject the batch."""
    bt = Batch(104, 30, 16, 2, 3, 2).device()
    QtT, Qaux = mvk.batch_preprocess([k.Q for k in bt.keys], bt.dc2)
    Ut = host(mvk.batch_project(QtT, bt.n, dev(bt.ei), dev(bt.ev)))
    bad = bt.Y.copy()
    bad[0, 2] = (int(bad[0, 2]) + 1000) % P
    inv_x = pow(int(bt.X[0, 0]), P - 2, P)
    for q in range(bt.ei.shape[0]):
        e = np.zeros(bt.cy["N"], dtype=np.uint32)
        e[bt.ei[q]] = bt.ev[q]
        Ut[q, 0] = (int(Ut[q, 0]) + 1000 * int(oracle.syn(bt.cy, e)[2]) * inv_x) % P
    vL = torch.empty((2, 2), dtype=torch.int32, device="cuda")
    vR = torch.empty_like(vL)
    acc, vL, vR, _, _ = mvk.batch_verify(bt.dcy, bt.dc2, Qaux, dev(bt.X), dev(bad), dev(bt.ei), dev(bt.ev), dev(Ut),
                                         dev(bt.e2i), dev(bt.e2v), vL=vL, vR=vR)
    assert torch.equal(vL, vR)  # the original checks all pass
    assert host(acc).tolist() == [0, 0]
