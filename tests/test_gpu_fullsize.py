"""Full-size bit-exact parity at the LLM-layer shapes, every output whole.

11008 x 4096 with 16 query columns (r = 3, t_x = 64) and 28672 x 8192 with 64
columns (r = 4, t_x = 128), t_y = 31, ell = 2.  Against the oracle (threaded
over row and column blocks on the host's cores): P^T and Q of Preprocess, X^
of Encrypt, Y^ of the server product with the row-major and with the packed
weights, Y, v_L, v_R and the accept bits of Verify + Decrypt (one-call and
prepared paths), honest and with tampered responses (Protocol pvMVMD,
Sec. 6.1; completeness and soundness, Thm. 6.1).
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import Instance

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_10264_amd as mvk
    mvk._lib.load()


def _say(*a):
    print(*a, flush=True)


def hv(t: torch.Tensor) -> np.ndarray:
    """Device int32 field array -> host uint32 view (no extra copy)."""
    return t.cpu().numpy().view(np.uint32)


import paper_2609_10264_amd as mvk  # noqa: E402


def _full_layer(name):
    cfg = synth.CONFIGS[name]
    m, n, B, ell = cfg["m"], cfg["n"], cfg["B"], cfg["ell"]
    T = oracle.threads()
    _say(f"{name}: full compare m={m} n={n} B={B} with {T} oracle threads")
    inst = Instance(cfg["cid"], m, n, B, cfg["r"], cfg["tx"], cfg["ty"], ell).to_device()
    mvk.keygen(inst.key, inst.dW)
    PT, Q = oracle.keygen(inst.W, inst.cx, inst.cy, nthreads=T)
    assert np.array_equal(hv(inst.key.PT), PT), "P^T"
    assert np.array_equal(hv(inst.key.Q), Q), "Q"

    dXh = mvk.encode(inst.key, inst.dX, inst.dexi, inst.dexv)
    Xh = oracle.encode(inst.cx, inst.X, inst.exi, inst.exv)
    assert np.array_equal(hv(dXh), Xh), "X^"

    Yh = oracle.server_eval(inst.W, Xh, nthreads=T)
    dYh = mvk.server_eval(inst.dW, dXh)
    assert np.array_equal(hv(dYh), Yh), "Y^ (row-major W)"
    Wp = mvk.pack_weights(inst.dW)
    dYh_p = mvk.server_eval(Wp, dXh)
    assert np.array_equal(hv(dYh_p), Yh), "Y^ (packed W)"

    # one tampered column beside the honest ones: the oracle's verdict, values and decryption
    bad = Yh.copy()
    bcol, pos = B // 2, m - 3
    bad[bcol, pos] = (int(bad[bcol, pos]) + 987654) % synth.P
    prep = mvk.client_prepare(inst.key, inst.dexi, inst.dexv, inst.deyi, inst.deyv)
    Xh2 = mvk.encode_masked(inst.key, inst.dX, prep)
    assert torch.equal(Xh2, dXh), "masked encode"
    for resp in (Yh, bad):
        oacc, ovL, ovR = oracle.verify(inst.cy, Q, Xh, resp, inst.eyi, inst.eyv)
        Yo = oracle.decode(PT, resp, inst.exi, inst.exv, nthreads=T)
        dresp = torch.from_numpy(resp.view(np.int32)).cuda()
        vL = torch.empty((ell, B), dtype=torch.int32, device="cuda")
        vR = torch.empty_like(vL)
        Y, acc, _, _ = mvk.decode_verify(inst.key, dXh, dresp, inst.dexi, inst.dexv, inst.deyi, inst.deyv,
                                         vL=vL, vR=vR)
        assert np.array_equal(hv(vL), ovL) and np.array_equal(hv(vR), ovR), "v_L, v_R"
        assert hv(acc).tolist() == oacc.astype(np.uint32).tolist(), "accept"
        assert np.array_equal(hv(Y), Yo), "Y"
        vL2, vR2 = torch.empty_like(vL), torch.empty_like(vL)
        Y2, acc2, _, _ = mvk.decode_verify_masked(inst.key, dXh, dresp, prep, vL=vL2, vR=vR2)
        for a, b in ((Y2, Y), (acc2, acc), (vL2, vL), (vR2, vR)):
            assert torch.equal(a, b), "prepared path"
    want = [True] * B
    want[bcol] = False
    assert oracle.verify(inst.cy, Q, Xh, bad, inst.eyi, inst.eyv)[0].tolist() == want
    assert np.array_equal(oracle.decode(PT, Yh, inst.exi, inst.exv, nthreads=T),
                          oracle.server_eval(inst.W, inst.X, nthreads=T)), "completeness"


def test_mlp_up_11008x4096_full():
    _full_layer("mlp_up_11008x4096")


def test_mlp_large_28672x8192_full():
    _full_layer("mlp_large_28672x8192")
