"""The seeded sampling of the method's random draws (the paper leaves the
generator open; the library and the oracle each implement one written
specification, stated in include/mvk.h and in oracle/mvk_oracle.c).

Pins of the oracle's sampler against facts that do not come from it:
SplitMix64's published reference outputs, the distributions the paper asks
for (App. B: uniform permutations and diagonals over F_p^*; Sec. 3 and
Lemma 5.1: E_t^N has exactly t distinct positions, uniform support, values
uniform in F_p^*), and Lemma 5.1's exact acceptance probability with
challenges drawn this way.  Then the library's host sampler against the
oracle's, array for array.  CPU only.
"""
import ctypes
import math
import os
from collections import Counter

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
FIELDS = [synth.P, synth.P_BABYBEAR]


@pytest.fixture(params=FIELDS, ids=["m31", "babybear"])
def p(request):
    return request.param


def _mvk():
    from paper_2609_10264_amd import _lib as L
    if not os.path.exists(L.LIB_PATH) or not os.path.exists(L.LIB_PATH_BB):
        pytest.skip("libmvk.so / libmvk_bb.so not built (run __graft_entry__.build())")
    import paper_2609_10264_amd as mvk
    return mvk


def _chi2_ok(counts, cells, n, z=6.0):
    """Chi-square statistic of `counts` over `cells` equiprobable cells against
    its mean (cells - 1) plus z standard deviations (sqrt(2 (cells - 1)))."""
    exp = n / cells
    stat = sum((counts.get(c, 0) - exp) ** 2 / exp for c in range(cells))
    return stat < (cells - 1) + z * math.sqrt(2 * (cells - 1)), stat


def test_generator_matches_published_reference_outputs():
    vals = [int(line) for line in open(os.path.join(GOLDEN, "splitmix64_state1234567.txt"))
            if line.strip() and not line.startswith("#")]
    assert oracle.sm64_draws(1234567, len(vals)) == vals


def test_tags_are_the_ascii_names():
    mvk = _mvk()
    for name, text in (("TAG_CODE_X", b"mvk-codx"), ("TAG_CODE_Y", b"mvk-cody"), ("TAG_NOISE", b"mvk-nois"),
                       ("TAG_CHALLENGE", b"mvk-chal")):
        assert getattr(oracle, name) == getattr(mvk, name) == int.from_bytes(text, "big")


def test_code_permutations_are_uniform(p):
    """Fisher-Yates over N = 4: all 24 permutations, equally often."""
    n = 24 * 200
    seen = Counter()
    index = {}
    for s in range(n):
        c = oracle.sample_code(2, 2, s, oracle.TAG_CODE_X, p=p)
        for perm in (c["pi1"], c["pi2"]):
            key = tuple(int(x) for x in perm)
            assert sorted(key) == [0, 1, 2, 3]
            seen[index.setdefault(key, len(index))] += 1
    assert len(index) == 24
    ok, stat = _chi2_ok(seen, 24, 2 * n)
    assert ok, stat


def test_code_diagonals_are_uniform_over_nonzero_elements(p):
    c = oracle.sample_code(4096, 4, 7, oracle.TAG_CODE_Y, p=p)
    v = np.concatenate([c["v1"], c["v2"]]).astype(np.int64)
    assert v.min() >= 1 and v.max() <= p - 1
    counts = Counter((v * 16 // p).tolist())
    ok, stat = _chi2_ok(counts, 16, v.size)
    assert ok, stat
    # the permutations are permutations
    assert np.array_equal(np.sort(c["pi1"]), np.arange(c["N"])) and np.array_equal(np.sort(c["pi2"]), np.arange(c["N"]))


def test_sparse_support_is_a_uniform_subset(p):
    """E_t^N with N = 6, t = 2: t distinct positions; each of the 15 subsets
    equally often; values in [1, p-1]."""
    count = 15 * 300
    idx, val = oracle.sample_sparse(count, 6, 2, 99, oracle.TAG_NOISE, p=p)
    assert (idx[:, 0] != idx[:, 1]).all() and idx.max() < 6
    assert val.min() >= 1 and val.max() <= p - 1
    subsets = {s: i for i, s in enumerate((a, b) for a in range(6) for b in range(a + 1, 6))}
    counts = Counter(subsets[tuple(sorted(map(int, r)))] for r in idx)
    ok, stat = _chi2_ok(counts, 15, count)
    assert ok, stat


def test_sparse_full_support_and_edge_sizes(p):
    idx, val = oracle.sample_sparse(3, 7, 7, 5, oracle.TAG_CHALLENGE, p=p)
    for r in idx:
        assert sorted(r.tolist()) == list(range(7))
    idx, _ = oracle.sample_sparse(4, 1, 1, 5, oracle.TAG_CHALLENGE, p=p)
    assert idx.tolist() == [[0]] * 4
    # different tags and seeds give different streams
    a, _ = oracle.sample_sparse(1, 1 << 20, 8, 5, oracle.TAG_NOISE, p=p)
    b, _ = oracle.sample_sparse(1, 1 << 20, 8, 5, oracle.TAG_CHALLENGE, p=p)
    c, _ = oracle.sample_sparse(1, 1 << 20, 8, 6, oracle.TAG_NOISE, p=p)
    assert not np.array_equal(a, b) and not np.array_equal(a, c)


@pytest.mark.parametrize("k,r,seed", [(1, 1, 0), (5, 2, 1), (256, 2, 2609), (4096, 3, 2**63 + 5), (3000, 8, 77)])
def test_library_code_sampler_equals_oracle(k, r, seed, p):
    mvk = _mvk()
    for tag in (oracle.TAG_CODE_X, oracle.TAG_CODE_Y):
        a = mvk.sample_code(k, r, seed, tag, p=p)
        b = oracle.sample_code(k, r, seed, tag, p=p)
        for name in ("pi1", "pi2", "v1", "v2"):
            assert np.array_equal(a[name], b[name]), (name, tag)


@pytest.mark.parametrize("count,N,t,seed", [(1, 1, 1, 3), (8, 12288, 64, 4), (64, 32768, 128, 2**64 - 2),
                                            (2, 114688, 31, 11), (5, 40, 40, 12), (16, 512, 8, 13)])
def test_library_sparse_sampler_equals_oracle(count, N, t, seed, p):
    mvk = _mvk()
    for tag in (oracle.TAG_NOISE, oracle.TAG_CHALLENGE):
        a = mvk.sample_sparse(count, N, t, seed, tag, p=p)
        b = oracle.sample_sparse(count, N, t, seed, tag, p=p)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


@pytest.mark.parametrize("t", [1, 2])
def test_acceptance_probability_lemma_with_library_challenges(t, p):
    """Lemma 5.1 with the challenges the library draws: a response off by a
    Delta whose encoding has weight w is accepted with probability exactly
    C(N - w, t) / C(N, t) (up to 1/(p-1)).  Identity code, r = 1: Delta = e_i
    encodes to a vector supported on positions >= i, so w = N - i."""
    mvk = _mvk()
    N, i = 12, 5
    code = synth.identity_code(N, 1)
    W = np.eye(N, dtype=np.int8)
    _, Q = oracle.keygen(W, code, code, want_P=False, p=p)
    Xh = synth.field_uniform(1, (1, N), p=p)
    Yh = oracle.server_eval(W, Xh, p=p)
    bad = Yh.copy()
    bad[0, i] = (int(bad[0, i]) + 17) % p
    w = N - i
    trials = 6000
    eyi, eyv = mvk.sample_sparse(trials, N, t, 4242 + t, mvk.TAG_CHALLENGE, p=p)
    hits = 0
    for s in range(trials):
        acc, _, _ = oracle.verify(code, Q, Xh, bad, eyi[s:s + 1], eyv[s:s + 1], p=p)
        hits += int(acc[0])
    prob = math.comb(N - w, t) / math.comb(N, t)
    sd = math.sqrt(prob * (1 - prob) / trials)
    assert abs(hits / trials - prob) < 5 * sd + 1e-9


def test_library_sampler_argument_checks():
    mvk = _mvk()
    from paper_2609_10264_amd import _lib as L
    lib = L.load()
    buf = (ctypes.c_uint32 * 8)()
    assert lib.mvk_sample_sparse(1, 4, 5, 0, 0, buf, buf) == L.MVK_EINVAL  # t > N
    assert lib.mvk_sample_sparse(1, 4, 2, 0, 0, None, buf) == L.MVK_EINVAL
    assert lib.mvk_sample_sparse(0, 4, 2, 0, 0, None, None) == L.MVK_OK
    assert lib.mvk_sample_code(0, 2, 0, 0, buf, buf, buf, buf) == L.MVK_EINVAL
    assert lib.mvk_sample_code(1 << 16, 1 << 16, 0, 0, buf, buf, buf, buf) == L.MVK_ERANGE
    assert mvk.sample_sparse(2, 10, 3, 1, mvk.TAG_NOISE)[0].shape == (2, 3)
