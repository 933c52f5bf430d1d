"""The allocation-free server product (mvk_server_eval_packed_static) against
mvk_server_eval_packed, through the C ABI, bit for bit: two calls in a row,
the second on a smaller input (the static scratch keeps the first call's
contents, so the second must not depend on them), then a shape without
scratch.  (The size limit is checked on the host, in test_abi.py.)"""
import ctypes

import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _run(fn_name, Wp, m, n, X, B):
    import paper_2609_10264_amd as mvk
    L = mvk._lib.load()
    Y = torch.full((B, m), -1, dtype=torch.int32, device="cuda")
    st = getattr(L, fn_name)(Wp.data.data_ptr(), m, n, X.data_ptr(), B, Y.data_ptr(), _stream())
    assert st == 0, (fn_name, st)
    return Y


@pytest.mark.parametrize("shapes", [
    # (m, n, B): large scratch first, then smaller ones
    [(28672, 8192, 64), (11008, 4096, 16), (4096, 4096, 8)],
    [(3001, 4160, 40), (257, 1000, 6), (4096, 4096, 1)],
])
def test_static_matches_workspace_entry_point(shapes):
    import paper_2609_10264_amd as mvk
    for i, (m, n, B) in enumerate(shapes):
        print(f"static server_eval call {i}: m={m} n={n} B={B}", flush=True)
        W = torch.randint(-127, 128, (m, n), dtype=torch.int8, device="cuda",
                          generator=torch.Generator(device="cuda").manual_seed(100 + i))
        Wp = mvk.pack_weights(W)
        X = torch.from_numpy(synth.field_uniform(200 + i, (B, n)).astype(np.int32)).cuda()
        want = _run("mvk_server_eval_packed", Wp, m, n, X, B)
        got = _run("mvk_server_eval_packed_static", Wp, m, n, X, B)
        torch.cuda.synchronize()
        assert torch.equal(got, want), (m, n, B)
