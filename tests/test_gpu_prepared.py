"""GPU parity of the prepared (boost / pipelined standard mode) path and the
stream flags: client_prepare, encode_masked and decode_verify_masked against
the oracle and against the one-call path, bit-exact."""
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


def _dense(N, idx, val):
    e = np.zeros(N, dtype=np.uint32)
    e[idx] = val
    return e


# cid, m, n, B, r_x, r_y, t_x, ell: block lengths in the one-launch range and
# above it (Nx = 16500, Ny = 18000: the syndromes take their own launches),
# several noise vectors and challenges, ragged column blocks of the 4-byte
# gathers (64 columns per item: up to 1024 items, or m, n not multiples of 4)
# and of the 16-byte ones (95, 96: 256 columns per item; 97: the separate
# gather launch with 1024-column items, ragged in m and n).
PREP = [
    (80, 256, 256, 1, 2, 2, 8, 2),
    (81, 1000, 700, 3, 3, 2, 17, 3),
    (82, 4096, 4096, 1, 3, 3, 64, 2),
    (83, 300, 5500, 2, 3, 3, 64, 2),
    (84, 6000, 200, 1, 1, 3, 5, 16),
    (85, 1001, 703, 3, 3, 2, 17, 3),
    (95, 1000, 300, 70, 2, 2, 9, 2),
    (96, 2048, 1000, 40, 2, 2, 9, 3),
    (97, 11008, 4100, 32, 2, 2, 16, 2),
]


@pytest.mark.parametrize("cid,m,n,B,rx,ry,tx,ell", PREP)
def test_client_prepare_matches_oracle(cid, m, n, B, rx, ry, tx, ell):
    _say(f"client_prepare cid={cid} m={m} n={n} B={B} rx={rx} ry={ry} tx={tx} ell={ell}")
    inst = Instance(cid, m, n, B, rx, tx, ty=31, ell=ell, ry=ry).to_device()
    mvk.keygen(inst.key, inst.dW)
    prep = mvk.client_prepare(inst.key, inst.dexi, inst.dexv, inst.deyi, inst.deyv)
    torch.cuda.synchronize()
    # input masks: Encrypt of the zero query
    Mx = oracle.encode(inst.cx, np.zeros((B, n), dtype=np.uint32), inst.exi, inst.exv)
    assert np.array_equal(host(prep.Mx), Mx)
    # output masks: P e = W (Gx e), since P = W Gx
    assert np.array_equal(host(prep.My), oracle.server_eval(inst.W, Mx))
    # challenge syndromes and u_q = e_q^T Q = (Gy e_q)^T W, since Q = Gy^T W
    R = np.stack([oracle.syn(inst.cy, _dense(inst.cy["N"], inst.eyi[q], inst.eyv[q])) for q in range(ell)])
    assert np.array_equal(host(prep.R), R)
    assert np.array_equal(host(prep.U), oracle.server_eval(np.ascontiguousarray(inst.W.T), R))


# few-workgroup decode/verify (B * (m + n) <= 32768 and ell <= 4: four
# elements per thread, one workgroup up to 4096 elements, three for 12000;
# ell 2 and 3),
# the element-block x column-group kernel above that (ell <= 4; one element
# per thread and 4 / ell columns per workgroup, or at 256 workgroups and more
# four elements and 16 / ell columns; ragged column groups and element blocks,
# n > m) and the general kernel (ell = 7); the segment kernel (above 4096
# elements, up to 8 columns with ell <= 2, 4 with ell <= 4): 8 columns in 17
# segments of one element per thread (110), 5 columns, ell = 1, n > m in 22
# segments of two (111), ell = 4 and 3 columns in 20 segments of four (112),
# ell = 3 and 2 columns in 40 segments (113), one column (114), all ragged
MASKED = PREP[:2] + PREP[3:4] + PREP[6:] + [(86, 3000, 2000, 8, 2, 2, 16, 3), (87, 500, 400, 2, 2, 2, 9, 7),
                                 (88, 12000, 300, 2, 2, 2, 9, 2), (90, 4096, 1000, 20, 2, 2, 16, 2),
                                 (91, 700, 5000, 13, 2, 2, 9, 4), (92, 1500, 1500, 9, 2, 2, 9, 1),
                                 (93, 16384, 100, 128, 2, 2, 5, 2), (94, 16000, 90, 64, 2, 2, 5, 3),
                                 (110, 4100, 4096, 8, 3, 3, 64, 2), (111, 4100, 11008, 5, 2, 2, 16, 1),
                                 (112, 20000, 300, 3, 2, 2, 9, 4), (113, 40000, 1000, 2, 2, 2, 9, 3),
                                 (114, 33000, 500, 1, 2, 2, 9, 2)]


@pytest.mark.parametrize("cid,m,n,B,rx,ry,tx,ell", MASKED)
def test_masked_path_matches_one_call_path(cid, m, n, B, rx, ry, tx, ell):
    _say(f"masked path cid={cid} m={m} n={n} B={B}")
    inst = Instance(cid, m, n, B, rx, tx, ty=31, ell=ell, ry=ry).to_device()
    mvk.keygen(inst.key, inst.dW)
    PT, Q = oracle.keygen(inst.W, inst.cx, inst.cy)
    prep = mvk.client_prepare(inst.key, inst.dexi, inst.dexv, inst.deyi, inst.deyv)
    Xh = mvk.encode_masked(inst.key, inst.dX, prep)
    Xh_ref = oracle.encode(inst.cx, inst.X, inst.exi, inst.exv)
    assert np.array_equal(host(Xh), Xh_ref)
    Yh = oracle.server_eval(inst.W, Xh_ref)
    bad = Yh.copy()
    bad[B - 1, m // 2] = (int(bad[B - 1, m // 2]) + 12345) % P
    for resp, want in ((Yh, [1] * B), (bad, [1] * (B - 1) + [0])):
        vL = torch.empty((ell, B), dtype=torch.int32, device="cuda")
        vR = torch.empty_like(vL)
        Y, acc, vL, vR = mvk.decode_verify_masked(inst.key, Xh, dev(resp), prep, vL=vL, vR=vR)
        oacc, ovL, ovR = oracle.verify(inst.cy, Q, Xh_ref, resp, inst.eyi, inst.eyv)
        assert oacc.astype(np.uint32).tolist() == want
        assert host(acc).tolist() == want
        assert np.array_equal(host(vL), ovL) and np.array_equal(host(vR), ovR)
        assert np.array_equal(host(Y), oracle.decode(PT, resp, inst.exi, inst.exv))
    # in place: Xhat may be X's own buffer
    Xc = inst.dX.clone()
    mvk.encode_masked(inst.key, Xc, prep, out=Xc)
    assert np.array_equal(host(Xc), Xh_ref)


def test_flags_order_two_streams():
    flags = torch.zeros(4, dtype=torch.int32, device="cuda")
    late = torch.zeros(1, dtype=torch.int32, device="cuda")[0]
    buf = torch.zeros(1 << 20, dtype=torch.int32, device="cuda")
    side, main = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    # the data written before the signal is seen after the wait (the signalling
    # stream's work is submitted first: the two streams may share a hardware queue)
    with torch.cuda.stream(side):
        buf.fill_(3)
        mvk.flag_signal(flags[0], 7, stream=side)
    mvk.flag_wait(flags[0], 7, timeout_us=2_000_000, timed_out=late, stream=main)
    with torch.cuda.stream(main):
        total = buf.to(torch.int64).sum()
    torch.cuda.synchronize()
    assert int(late.item()) == 0
    assert int(total.item()) == 3 * buf.numel()
    assert int(flags[0].item()) == 0  # the wait consumed the signal
    # a wait that is never signalled ends after its time-out and says so
    mvk.flag_wait(flags[1], 5, timeout_us=2000, timed_out=late, stream=main)
    torch.cuda.synchronize()
    assert int(late.item()) == 1 and int(flags[1].item()) == 0


def test_flags_order_compute_unit_streams():
    """Two streams on disjoint compute-unit ranges (mvk_stream_create_cu_range):
    a flag wait on one sees the data the other wrote before its signal, and a
    server product on a restricted stream equals the one on a plain stream;
    a range past the device's units is refused."""
    ncu = mvk.device_cus()
    with pytest.raises(mvk.MvkError):
        mvk.CUStream(ncu - 4, 8)
    a, b = mvk.CUStream(0, 64), mvk.CUStream(64, ncu - 64)
    try:
        flag = torch.zeros((), dtype=torch.int32, device="cuda")
        late = torch.zeros((), dtype=torch.int32, device="cuda")
        buf = torch.zeros(1 << 20, dtype=torch.int32, device="cuda")
        torch.cuda.synchronize()
        with torch.cuda.stream(a.stream):
            buf.fill_(5)
            mvk.flag_signal(flag, 3, stream=a.stream)
        mvk.flag_wait(flag, 3, timeout_us=2_000_000, timed_out=late, stream=b.stream)
        with torch.cuda.stream(b.stream):
            total = buf.to(torch.int64).sum()
        torch.cuda.synchronize()
        assert int(late.item()) == 0 and int(flag.item()) == 0
        assert int(total.item()) == 5 * buf.numel()
        W = dev(synth.weights(synth.seed_for(62, synth.PURPOSE_W), 1000, 700))
        X = dev(synth.field_uniform(synth.seed_for(62, synth.PURPOSE_X), (8, 700)))
        ref = mvk.server_eval(W, X)
        with torch.cuda.stream(a.stream):
            ya = mvk.server_eval(W, X, stream=a.stream)
        torch.cuda.synchronize()
        assert torch.equal(ya, ref)
    finally:
        a.close()
        b.close()
    # destroying a stream retires its workspace: streams created afterwards
    # (which may get the same handle) start with a fresh one, and the
    # retired buffers are freed by mvk_workspace_release
    for _ in range(2):
        c = mvk.CUStream(0, ncu)
        try:
            with torch.cuda.stream(c.stream):
                yc = mvk.server_eval(mvk.pack_weights(W), X, stream=c.stream)
            torch.cuda.synchronize()
            assert torch.equal(yc, ref)
        finally:
            c.close()
    assert mvk._lib.load().mvk_workspace_release() == 0


@pytest.mark.parametrize("cid,m,n,B,r,tx,ell", [(98, 4096, 4096, 1, 3, 64, 2), (99, 1000, 700, 3, 3, 17, 3),
                                                (100, 3000, 2000, 8, 2, 16, 2), (101, 12000, 300, 2, 2, 9, 2)])
def test_client_turn_matches_two_calls(cid, m, n, B, r, tx, ell):
    """decode_verify_encode_masked (the decode/verify of one response and the
    masked encode of the next query in one launch; 12000 x 300, B = 2: three
    decode/verify workgroups; 3000 x 2000, B = 8: the two-launch form) gives
    the outputs of
    decode_verify_masked and encode_masked, with a tampered column rejected;
    and a turn whose next query waits for a flag set on another stream."""
    print(f"client turn cid={cid} m={m} n={n} B={B} ell={ell}", flush=True)
    inst = Instance(cid, m, n, B, r, tx, ty=31, ell=ell).to_device()
    mvk.keygen(inst.key, inst.dW)
    prep = mvk.client_prepare(inst.key, inst.dexi, inst.dexv, inst.deyi, inst.deyv)
    nxt = Instance(cid + 50, m, n, B, r, tx, ty=31, ell=ell).to_device()
    prep2 = mvk.client_prepare(inst.key, nxt.dexi, nxt.dexv, nxt.deyi, nxt.deyv)
    Xh = mvk.encode_masked(inst.key, inst.dX, prep)
    Yh = mvk.server_eval(inst.dW, Xh)
    Yh[B - 1, m // 3] = (Yh[B - 1, m // 3].to(torch.int64) + 99) % P
    vL, vR = (torch.empty((ell, B), dtype=torch.int32, device="cuda") for _ in range(2))
    Y, acc, _, _, Xh2 = mvk.decode_verify_encode_masked(inst.key, Xh, Yh, prep, nxt.dX, prep2, vL=vL, vR=vR)
    vL1, vR1 = (torch.empty((ell, B), dtype=torch.int32, device="cuda") for _ in range(2))
    Y1, acc1, _, _ = mvk.decode_verify_masked(inst.key, Xh, Yh, prep, vL=vL1, vR=vR1)
    Xh21 = mvk.encode_masked(inst.key, nxt.dX, prep2)
    torch.cuda.synchronize()
    for a, b in ((Y, Y1), (acc, acc1), (vL, vL1), (vR, vR1), (Xh2, Xh21)):
        assert torch.equal(a, b)
    assert host(acc).tolist() == [1] * (B - 1) + [0]
    # the next query's mask prepared on another stream, ordered by a flag
    flag = torch.zeros((), dtype=torch.int32, device="cuda")
    late = torch.zeros((), dtype=torch.int32, device="cuda")
    side, main = torch.cuda.Stream(), torch.cuda.Stream()
    prep3 = mvk.Prepared(inst.key, B, ell)
    torch.cuda.synchronize()
    with torch.cuda.stream(side):
        mvk.client_prepare(inst.key, nxt.dexi, nxt.dexv, nxt.deyi, nxt.deyv, out=prep3, done_flag=flag,
                           stream=side)
    with torch.cuda.stream(main):
        _, _, _, _, Xh3 = mvk.decode_verify_encode_masked(inst.key, Xh, Yh, prep, nxt.dX, prep3, ready_flag=flag,
                                                         timeout_us=2_000_000, timed_out=late, stream=main)
    torch.cuda.synchronize()
    assert int(late.item()) == 0 and int(flag.item()) == 0
    assert torch.equal(Xh3, Xh21)


def test_pipelined_graphs_match_one_call_path():
    """The pipelined standard mode as two HIP graphs (preparation stream ahead of
    the online stream, ordered by flags) against the one-call path, per step."""
    cid, m, n, B, r, tx, ell, steps = 85, 1000, 700, 2, 3, 17, 2, 4
    inst = Instance(cid, m, n, B, r, tx, ty=31, ell=ell).to_device()
    mvk.keygen(inst.key, inst.dW)
    exi, exv = synth.sparse(synth.seed_for(cid, synth.PURPOSE_NOISE, 1), steps * B, inst.cx["N"], tx)
    eyi, eyv = synth.sparse(synth.seed_for(cid, synth.PURPOSE_CHAL, 1), steps * ell, inst.cy["N"], 31)
    EXI, EXV = dev(exi).view(steps, B, tx), dev(exv).view(steps, B, tx)
    EYI, EYV = dev(eyi).view(steps, ell, 31), dev(eyv).view(steps, ell, 31)
    X = dev(synth.field_uniform(synth.seed_for(cid, synth.PURPOSE_X, 1), (steps, B, n)))
    preps = [mvk.Prepared(inst.key, B, ell) for _ in range(steps)]
    flags = torch.zeros(steps, dtype=torch.int32, device="cuda")
    late = torch.zeros((), dtype=torch.int32, device="cuda")
    Xh = torch.empty((steps, B, n), dtype=torch.int32, device="cuda")
    Yh = torch.empty((steps, B, m), dtype=torch.int32, device="cuda")
    Y = torch.empty((steps, B, m), dtype=torch.int32, device="cuda")
    acc = torch.zeros((steps, B), dtype=torch.int32, device="cuda")
    side, main = torch.cuda.Stream(), torch.cuda.Stream()

    def prepare(i):  # odd steps: the flag kernels; even steps: the flags fused into the calls
        if i % 2:
            mvk.client_prepare(inst.key, EXI[i], EXV[i], EYI[i], EYV[i], out=preps[i])
            mvk.flag_signal(flags[i], 1)
        else:
            mvk.client_prepare(inst.key, EXI[i], EXV[i], EYI[i], EYV[i], out=preps[i], done_flag=flags[i])

    def online(i):
        if i % 2:
            mvk.flag_wait(flags[i], 1, timeout_us=500_000, timed_out=late)
            mvk.encode_masked(inst.key, X[i], preps[i], out=Xh[i])
        else:
            mvk.encode_masked(inst.key, X[i], preps[i], out=Xh[i], ready_flag=flags[i], timeout_us=500_000,
                              timed_out=late)
        mvk.server_eval(inst.dW, Xh[i], out=Yh[i])
        mvk.decode_verify_masked(inst.key, Xh[i], Yh[i], preps[i], Y=Y[i], accept=acc[i])

    for s, fn in ((side, prepare), (main, online)):  # size the per-stream workspaces outside capture
        with torch.cuda.stream(s):
            fn(0)
    torch.cuda.synchronize()
    gp, go = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.graph(gp, stream=side):
        for i in range(steps):
            prepare(i)
    with torch.cuda.graph(go, stream=main):
        for i in range(steps):
            online(i)
    for rep in range(2):
        Y.zero_()
        acc.zero_()
        torch.cuda.synchronize()
        with torch.cuda.stream(side):  # the preparation graph is submitted first
            gp.replay()
        with torch.cuda.stream(main):
            go.replay()
        torch.cuda.synchronize()
        assert int(late.item()) == 0, rep
        assert host(acc).tolist() == [[1] * B] * steps
        for i in range(steps):
            Xr = mvk.encode(inst.key, X[i], EXI[i], EXV[i])
            Yr = mvk.server_eval(inst.dW, Xr)
            Yd, accr, _, _ = mvk.decode_verify(inst.key, Xr, Yr, EXI[i], EXV[i], EYI[i], EYV[i])
            assert torch.equal(Xh[i], Xr) and torch.equal(Yh[i], Yr) and torch.equal(Y[i], Yd), (rep, i)
        assert host(flags).tolist() == [0] * steps


@pytest.mark.parametrize("cid,m,n,B,ry,ell", [(90, 256, 256, 1, 2, 2), (91, 1000, 700, 3, 3, 5), (92, 6000, 300, 2, 3, 2)])
def test_verify_only_mode(cid, m, n, B, ry, ell):
    """Verification without privacy: plaintext queries and results, accepted
    when Y = W X, rejected column by column when a result is changed."""
    _say(f"verify only cid={cid} m={m} n={n} B={B}")
    inst = Instance(cid, m, n, B, 2, 0, ty=31, ell=ell, ry=ry).to_device()
    mvk.keygen(inst.key, inst.dW)
    _, Q = oracle.keygen(inst.W, inst.cx, inst.cy, want_P=False)
    Yp = oracle.server_eval(inst.W, inst.X)
    bad = Yp.copy()
    bad[0, 3] = (int(bad[0, 3]) + 1) % P
    for resp, want in ((Yp, [1] * B), (bad, [0] + [1] * (B - 1))):
        vL = torch.empty((ell, B), dtype=torch.int32, device="cuda")
        vR = torch.empty_like(vL)
        acc, vL, vR = mvk.verify(inst.key, inst.dX, dev(resp), inst.deyi, inst.deyv, vL=vL, vR=vR)
        oacc, ovL, ovR = oracle.verify(inst.cy, Q, inst.X, resp, inst.eyi, inst.eyv)
        assert oacc.astype(np.uint32).tolist() == want == host(acc).tolist()
        assert np.array_equal(host(vL), ovL) and np.array_equal(host(vR), ovR)


# ---------------------------------------------------------------------------
# groups of keys sharing an input (one launch for several matrices)
# ---------------------------------------------------------------------------
def _group(G, m, n, B, r, tx, ty, ell, sub):
    cx = synth.raa_code(synth.seed_for(60, synth.PURPOSE_CX, sub), n, r)
    cy = synth.raa_code(synth.seed_for(60, synth.PURPOSE_CY, sub), m, r)
    dcx, dcy = code(cx), code(cy)
    Ws = [synth.weights(synth.seed_for(60, synth.PURPOSE_W, sub + g), m, n) for g in range(G)]
    keys = []
    for W in Ws:
        k = mvk.Key.allocate(m, n, dcx, dcy)
        mvk.keygen(k, dev(W))
        keys.append(k)
    exi, exv = synth.sparse(synth.seed_for(60, synth.PURPOSE_NOISE, sub), B, cx["N"], tx)
    eys = [tuple(dev(a) for a in synth.sparse(synth.seed_for(60, synth.PURPOSE_CHAL, sub + g), ell, cy["N"], ty))
           for g in range(G)]
    X = synth.field_uniform(synth.seed_for(60, synth.PURPOSE_X, sub), (B, n))
    return Ws, keys, dev(exi), dev(exv), eys, X


@pytest.mark.parametrize("G,m,n,B,r,tx,ell", [(3, 4096, 4096, 8, 3, 64, 2), (2, 11008, 4096, 8, 3, 64, 2),
                                              (3, 300, 200, 2, 2, 10, 3), (2, 6000, 6000, 3, 3, 40, 2),
                                              (4, 512, 640, 16, 2, 20, 4), (1, 1000, 900, 5, 3, 30, 2)])
def test_group_preparation_and_checks_match_one_key_at_a_time(G, m, n, B, r, tx, ell):
    """client_prepare_group and decode_verify_masked_group give, for every key,
    the outputs of client_prepare and decode_verify_masked, bit for bit, with a
    tampered response in the group."""
    print(f"group prepare/check G={G} m={m} n={n} B={B} ell={ell}", flush=True)
    Ws, keys, exi, exv, eys, X = _group(G, m, n, B, r, tx, 31, ell, 100 * G + m % 97)
    preps = mvk.client_prepare_group(keys, exi, exv, eys)
    singles = [mvk.client_prepare(k, exi, exv, *ey) for k, ey in zip(keys, eys)]
    for g in range(G):
        for name in ("Mx", "My", "R", "U"):
            assert torch.equal(getattr(preps[g], name), getattr(singles[g], name)), (g, name)
    Xh = mvk.encode_masked(keys[0], dev(X), preps[0])
    Yhs = [mvk.server_eval(dev(W), Xh) for W in Ws]
    Yhs[G - 1][B - 1, m // 2] = (Yhs[G - 1][B - 1, m // 2].to(torch.int64) + 31337) % P
    vLs = [torch.empty((ell, B), dtype=torch.int32, device="cuda") for _ in range(G)]
    vRs = [torch.empty_like(v) for v in vLs]
    Ys, accs, _, _ = mvk.decode_verify_masked_group(keys, Xh, Yhs, preps, vLs=vLs, vRs=vRs)
    for g in range(G):
        vL = torch.empty((ell, B), dtype=torch.int32, device="cuda")
        vR = torch.empty_like(vL)
        Y1, acc1, _, _ = mvk.decode_verify_masked(keys[g], Xh, Yhs[g], singles[g], vL=vL, vR=vR)
        for a, b in ((Ys[g], Y1), (accs[g], acc1), (vLs[g], vL), (vRs[g], vR)):
            assert torch.equal(a, b), g
        want = [1] * B
        if g == G - 1:
            want[B - 1] = 0
        assert host(accs[g]).tolist() == want, g
    # the honest outputs decrypt to W x (oracle); the tampered column is the last one of the last key
    assert np.array_equal(host(Ys[0])[:B - 1], oracle.server_eval(Ws[0], X)[:B - 1])


def test_multi_preparation_matches_oracle():
    """client_prepare_multi over six keys of four shapes and four inputs: two
    keys share an input (one noise, one privacy code), one input's noise
    syndrome and one key's challenge syndromes are longer than 16384 (their own
    launches), one key has no noise and one no challenges.  Every output
    against the oracle (masks by Encrypt of the zero query, P e = W Gx e,
    R by the syndrome, U = R^T W), and the done flags set."""
    print("multi prepare: six keys, four inputs", flush=True)
    # (m, n, r_x, r_y, t_x, ell, input), input None: no noise; ell 0: no challenges
    spec = [(1000, 700, 3, 2, 17, 3, 0), (1000, 700, 3, 3, 17, 2, 0), (6000, 200, 2, 3, 5, 2, 1),
            (300, 5500, 3, 2, 64, 2, 2), (2048, 1000, 2, 2, 9, 3, None), (512, 640, 2, 2, 20, 0, 3)]
    B = {0: 3, 1: 2, 2: 2, 3: 4}
    cxs, inputs = {}, {}
    keys, hosts, exs, eys = [], [], [], []
    for g, (m, n, rx, ry, tx, ell, inp) in enumerate(spec):
        sub = 900 + g
        W = synth.weights(synth.seed_for(61, synth.PURPOSE_W, sub), m, n)
        cxk = inp if inp is not None else ("own", g)
        if cxk not in cxs:
            c = synth.raa_code(synth.seed_for(61, synth.PURPOSE_CX, 500 + len(cxs)), n, rx)
            cxs[cxk] = (c, code(c))
        cx_h, cx_d = cxs[cxk]
        cy_h = synth.raa_code(synth.seed_for(61, synth.PURPOSE_CY, sub), m, ry)
        key = mvk.Key.allocate(m, n, cx_d, code(cy_h))
        mvk.keygen(key, dev(W))
        keys.append(key)
        if inp is not None and inp not in inputs:
            i_, v_ = synth.sparse(synth.seed_for(61, synth.PURPOSE_NOISE, inp), B[inp], cx_h["N"], tx)
            inputs[inp] = (i_, v_, (dev(i_), dev(v_)))
        exs.append(inputs[inp][2] if inp is not None else None)
        ey_h = synth.sparse(synth.seed_for(61, synth.PURPOSE_CHAL, sub), ell, cy_h["N"], 31) if ell else None
        eys.append(tuple(dev(a) for a in ey_h) if ell else None)
        hosts.append((W, cx_h, cy_h, inputs[inp][:2] if inp is not None else None, ey_h))
    assert cxs[0][0]["N"] <= 16384 < cxs[2][0]["N"] and spec[2][0] * spec[2][3] > 16384
    flags = [torch.zeros((), dtype=torch.int32, device="cuda") for _ in range(2)]
    done = [flags[g % 2] if g < 4 else None for g in range(len(spec))]
    preps = mvk.client_prepare_multi(keys, exs, eys, done_flags=done, done_value=7)
    torch.cuda.synchronize()
    assert [int(f.item()) for f in flags] == [7, 7]
    assert preps[0].Mx.data_ptr() == preps[1].Mx.data_ptr()
    for g, (W, cx_h, cy_h, ex_h, ey_h) in enumerate(hosts):
        m, n = W.shape
        if ex_h is not None:
            Bg = ex_h[0].shape[0]
            Mx = oracle.encode(cx_h, np.zeros((Bg, n), dtype=np.uint32), *ex_h)
            assert np.array_equal(host(preps[g].Mx), Mx), (g, "Mx")
            assert np.array_equal(host(preps[g].My), oracle.server_eval(W, Mx)), (g, "My")
        if ey_h is not None:
            R = np.stack([oracle.syn(cy_h, _dense(cy_h["N"], ey_h[0][q], ey_h[1][q])) for q in range(ey_h[0].shape[0])])
            assert np.array_equal(host(preps[g].R), R), (g, "R")
            assert np.array_equal(host(preps[g].U), oracle.server_eval(np.ascontiguousarray(W.T), R)), (g, "U")


# m, n, B, ell: the one-workgroup form (m != n: rejected), one workgroup per
# column (ell 2 and 4, 8 and 40 columns), segmented sums (ell 2 and 3), the
# element-block form (70000 rows: longer than one column's workgroup or
# segments take) and the general form (ell = 6)
MAXVAL = [(1000, 900, 2, 2), (4096, 4096, 8, 2), (4096, 4096, 8, 4), (3000, 3000, 40, 2), (12000, 12000, 4, 2),
          (12000, 11000, 3, 3), (70000, 1000, 1, 2), (70000, 1000, 3, 4), (2000, 2000, 3, 6)]


@pytest.mark.parametrize("m,n,B,ell", MAXVAL)
def test_decode_verify_masked_at_max_values_closed_form(m, n, B, ell):
    """Every input p - 1 (X^, Y^, the masks My and the challenge vectors R,
    U): (p - 1)^2 = 1 mod p, so v_L = n and v_R = m mod p in every column and
    repetition, Y = 0, and the columns are accepted exactly when m = n; the
    64-bit sums of every check kernel run at their largest terms."""
    _say(f"decode_verify_masked max values m={m} n={n} B={B} ell={ell}")
    cx = code(synth.raa_code(synth.seed_for(62, synth.PURPOSE_CX, n), n, 1))
    cy = code(synth.raa_code(synth.seed_for(62, synth.PURPOSE_CY, m), m, 1))
    key = mvk.Key.allocate(m, n, cx, cy)  # P^T and Q are not read by the masked check
    prep = mvk.Prepared(key, B, ell)
    for t in (prep.My, prep.R, prep.U, prep.Mx):
        t.fill_(P - 1)
    Xh = torch.full((B, n), P - 1, dtype=torch.int32, device="cuda")
    Yh = torch.full((B, m), P - 1, dtype=torch.int32, device="cuda")
    vL = torch.full((ell, B), -1, dtype=torch.int32, device="cuda")
    vR = torch.full_like(vL, -1)
    Y, acc, _, _ = mvk.decode_verify_masked(key, Xh, Yh, prep, vL=vL, vR=vR)
    torch.cuda.synchronize()
    assert not host(Y).any()
    assert (host(vL) == n % P).all() and (host(vR) == m % P).all()
    assert host(acc).tolist() == [1 if m == n else 0] * B
