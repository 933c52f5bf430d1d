"""The usage sequence of the library, as a user writes it: Preprocess,
Encrypt, server product, Decrypt + Verify, then the prepared (standard mode
with precomputation) calls, over both fields; the decrypted result is the
plaintext product and every column is accepted."""
import numpy as np
import pytest
import torch

import synth
from tests.gpu_util import dev, host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.parametrize("p", [synth.P, synth.P_BABYBEAR], ids=["m31", "babybear"])
def test_usage_sequence(p):
    import paper_2609_10264_amd as mvk

    m, n, B, r, tx, ty, ell = 300, 200, 3, 3, 9, 31, 2
    W = dev(synth.weights(71, m, n))
    X = dev(synth.field_uniform(72, (B, n), p=p))
    c = [synth.raa_code(73 + i, k, r, p=p) for i, k in enumerate((n, m))]
    cx, cy = (mvk.Code(x["k"], x["r"], dev(x["pi1"]), dev(x["pi2"]), dev(x["v1"]), dev(x["v2"]), p) for x in c)
    ex_idx, ex_val = (dev(a) for a in synth.sparse(75, B, r * n, tx, p=p))
    ey_idx, ey_val = (dev(a) for a in synth.sparse(76, ell, r * m, ty, p=p))

    key = mvk.keygen(mvk.Key.allocate(m, n, cx, cy), W)
    Wp = mvk.pack_weights(W)
    Xhat = mvk.encode(key, X, ex_idx, ex_val)
    Yhat = mvk.server_eval(Wp, Xhat, p=p)
    Y, accept, vL, vR = mvk.decode_verify(key, Xhat, Yhat, ex_idx, ex_val, ey_idx, ey_val)
    plain = host(mvk.server_eval(W, X, p=p))
    assert np.array_equal(host(Y), plain) and host(accept).tolist() == [1] * B

    prep = mvk.client_prepare(key, ex_idx, ex_val, ey_idx, ey_val)
    Xhat2 = mvk.encode_masked(key, X, prep)
    Y2, accept2, _, _ = mvk.decode_verify_masked(key, Xhat2, mvk.server_eval(Wp, Xhat2, p=p), prep)
    assert torch.equal(Xhat2, Xhat)
    assert np.array_equal(host(Y2), plain) and host(accept2).tolist() == [1] * B
