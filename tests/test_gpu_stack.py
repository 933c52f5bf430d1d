"""GPU parity of a 32-layer decoder stack delegated with pvMVMD.

Per layer: seven projections (q, k, v, o 4096x4096; up, gate 11008x4096; down
4096x11008), eight query columns, r = 3, t_x = 64, t_y = 31, ell = 2.  The
responses of a pass are enumerated (layer, projection, column); the one whose
index is congruent to a seeded offset modulo 1000 is tampered (a nonzero
delta at a seeded coordinate).

One test per layer compares, against the CPU oracle (threaded over the host's
cores), for every projection: the masked queries X^ in full, the responses Y^
in full, Q in full, v_L, v_R and the accept bits of Verify, and the
decrypted outputs Y.  On the first and last layer and on every layer that
holds a tampered response, P^T is compared whole too and Y with the
oracle's Decrypt; on the other layers Y is compared with W x, the oracle's
product of the plaintext (completeness, Thm. 6.1), which equals the oracle's
Decrypt of an honest response.  The prepared schedule (preparation stream,
flags, masked encode and decode/verify) must reproduce the one-call outputs.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import code as dev_code
from tests.gpu_util import dev

pytestmark = pytest.mark.gpu
P = synth.P
CFG = synth.STACK
LAYERS = int(os.environ.get("MVK_STACK_LAYERS", CFG["layers"]))


def hv(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint32)


@pytest.fixture(scope="module")
def stack_setup():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_10264_amd.stack as stack

    r, cid = CFG["r"], CFG["cid"]
    host_codes = {}

    def make_code(kind, k):
        purpose = synth.PURPOSE_CX if kind == "x" else synth.PURPOSE_CY
        c = synth.raa_code(synth.seed_for(cid, purpose, sub=k), k, r)
        host_codes[(kind, k)] = c
        return dev_code(c)

    cx_by_n, cy_by_m = stack.codes_for(make_code)
    nproj = len(stack.PROJECTIONS)
    total = CFG["layers"] * nproj * CFG["B"]
    g = synth.rng(synth.seed_for(cid, synth.PURPOSE_TAMPER))
    offset = int(g.integers(0, 1000))
    plan = {}  # (layer, projection index) -> [(column, coordinate, delta)]
    for k in range(offset, total, 1000):
        L, rest = divmod(k, nproj * CFG["B"])
        i, b = divmod(rest, CFG["B"])
        m = stack.PROJECTIONS[i][1]
        plan.setdefault((L, i), []).append((b, int(g.integers(0, m)), int(g.integers(1, P))))
    return stack, host_codes, cx_by_n, cy_by_m, plan, offset


def test_tamper_schedule_covers_a_pass(stack_setup):
    """One response in 1000 of the pass's 32 * 7 * 8 = 1792, at a seeded offset."""
    _, _, _, _, plan, offset = stack_setup
    total = CFG["layers"] * 7 * CFG["B"]
    assert sum(len(v) for v in plan.values()) == len(range(offset, total, 1000)) >= 1


@pytest.mark.parametrize("L", range(LAYERS))
def test_stack_layer_matches_oracle(stack_setup, L):
    stack, host_codes, cx_by_n, cy_by_m, plan, _ = stack_setup
    B, r, tx, ty, ell, cid = (CFG[k] for k in ("B", "r", "tx", "ty", "ell", "cid"))
    T = oracle.threads()
    print(f"stack layer {L} ({T} oracle threads)", flush=True)
    sub = 100 * (L + 1)
    Wh = {name: synth.weights(synth.seed_for(cid, synth.PURPOSE_W, sub + i), m, n)
          for i, (name, m, n, _) in enumerate(stack.PROJECTIONS)}
    layer = stack.build_layer({k: dev(v) for k, v in Wh.items()}, cx_by_n, cy_by_m)
    X_h, ex_h = {}, {}
    for j, grp in enumerate(stack.INPUTS):
        n = stack.input_width(grp)
        X_h[grp] = synth.field_uniform(synth.seed_for(cid, synth.PURPOSE_X, sub + j), (B, n))
        ex_h[grp] = synth.sparse(synth.seed_for(cid, synth.PURPOSE_NOISE, sub + j), B, r * n, tx)
    ey_h = {name: synth.sparse(synth.seed_for(cid, synth.PURPOSE_CHAL, sub + i), ell, r * m, ty)
            for i, (name, m, n, _) in enumerate(stack.PROJECTIONS)}
    X = {k: dev(v) for k, v in X_h.items()}
    ex = {k: (dev(a), dev(b)) for k, (a, b) in ex_h.items()}
    ey = {k: (dev(a), dev(b)) for k, (a, b) in ey_h.items()}
    mine = {stack.PROJECTIONS[i][0]: v for (LL, i), v in plan.items() if LL == L}

    def tamper(name, Yhat):
        for b, pos, delta in mine.get(name, []):
            Yhat[b, pos] = (Yhat[b, pos].to(torch.int64) + delta) % P

    out = stack.run_layer(layer, X, ex, ey, tamper=tamper)
    # the prepared schedule: the layer's preparation on its own stream (one
    # call, one flag), then the online part, whose first masked encode waits
    flag = torch.zeros((), dtype=torch.int32, device="cuda")
    late = torch.zeros((), dtype=torch.int32, device="cuda")
    s_prep, s_on = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s_prep):
        preps = stack.prepare_layer(layer, ex, ey, flag, stream=s_prep)
    with torch.cuda.stream(s_on):
        pout = stack.run_layer_prepared(layer, X, preps, ready_flag=flag, timeout_us=2_000_000, timed_out=late,
                                        tamper=tamper, stream=s_on)
    torch.cuda.synchronize()
    assert int(late.item()) == 0 and int(flag.item()) == 0
    for name in out:
        for a, b in zip(out[name], pout[name]):
            assert torch.equal(a, b), (L, name, "prepared schedule")

    full = L in (0, LAYERS - 1) or any(LL == L for (LL, _) in plan)
    Xh_o = {}
    for grp in stack.INPUTS:
        n = stack.input_width(grp)
        Xh_o[grp] = oracle.encode(host_codes[("x", n)], X_h[grp], *ex_h[grp])
    for i, (name, m, n, grp) in enumerate(stack.PROJECTIONS):
        cx, cy = host_codes[("x", n)], host_codes[("y", m)]
        Y, acc, Xh, Yh, vL, vR = out[name]
        key = layer.keys[name]
        assert np.array_equal(hv(Xh), Xh_o[grp]), (L, name, "X^")
        Yh_o = oracle.server_eval(Wh[name], Xh_o[grp], nthreads=T)
        for b, pos, delta in mine.get(name, []):
            Yh_o[b, pos] = (int(Yh_o[b, pos]) + delta) % P
        assert np.array_equal(hv(Yh), Yh_o), (L, name, "Y^")
        PT, Q = oracle.keygen(Wh[name], cx, cy, want_P=full, nthreads=T)
        assert np.array_equal(hv(key.Q), Q), (L, name, "Q")
        if full:
            assert np.array_equal(hv(key.PT), PT), (L, name, "P^T")
        oacc, ovL, ovR = oracle.verify(cy, Q, Xh_o[grp], Yh_o, *ey_h[name])
        assert np.array_equal(hv(vL), ovL) and np.array_equal(hv(vR), ovR), (L, name, "v_L, v_R")
        assert hv(acc).tolist() == oacc.astype(np.uint32).tolist(), (L, name, "accept")
        bad = {b for (b, _, _) in mine.get(name, [])}
        assert [b for b in range(B) if not oacc[b]] == sorted(bad), (L, name, "schedule")
        if full:
            assert np.array_equal(hv(Y), oracle.decode(PT, Yh_o, *ex_h[grp], nthreads=T)), (L, name, "Y")
        else:
            assert not bad
            assert np.array_equal(hv(Y), oracle.server_eval(Wh[name], X_h[grp], nthreads=T)), (L, name, "Y")
    del layer, out, pout, preps


def test_overlapped_pass_matches_one_call_path(stack_setup):
    """run_pass_overlapped (preparation streams one layer ahead, the projections
    of a stage on parallel branches) gives the one-call outputs bit for bit,
    eager and as a captured graph replayed three times with other work between
    the replays; a tampered response is rejected on both."""
    stack, _, cx_by_n, cy_by_m, _, _ = stack_setup
    import paper_2609_10264_amd as mvk

    B, r, tx, ty, ell, cid = (CFG[k] for k in ("B", "r", "tx", "ty", "ell", "cid"))
    nl = 3
    layers, inputs = [], []
    for L in range(nl):
        sub = 700 + 10 * L
        Ws = {name: dev(synth.weights(synth.seed_for(cid, synth.PURPOSE_W, sub + i), m, n))
              for i, (name, m, n, _) in enumerate(stack.PROJECTIONS)}
        layers.append(stack.build_layer(Ws, cx_by_n, cy_by_m))
        X = {g: dev(synth.field_uniform(synth.seed_for(cid, synth.PURPOSE_X, sub + j), (B, stack.input_width(g))))
             for j, g in enumerate(stack.INPUTS)}
        ex = {g: tuple(dev(a) for a in synth.sparse(synth.seed_for(cid, synth.PURPOSE_NOISE, sub + j), B,
                                                     r * stack.input_width(g), tx))
              for j, g in enumerate(stack.INPUTS)}
        ey = {name: tuple(dev(a) for a in synth.sparse(synth.seed_for(cid, synth.PURPOSE_CHAL, sub + i), ell,
                                                        r * m, ty))
              for i, (name, m, _, _) in enumerate(stack.PROJECTIONS)}
        inputs.append((X, ex, ey))

    def tamper(L, name, Yhat):
        if L == 1 and name == "up":
            Yhat[3, 100] = (Yhat[3, 100].to(torch.int64) + 5) % P

    ref = [stack.run_layer(layers[L], *inputs[L], tamper=lambda nm, Y, L=L: tamper(L, nm, Y)) for L in range(nl)]
    torch.cuda.synchronize()
    main = torch.cuda.Stream()
    preps_s = [torch.cuda.Stream() for _ in range(4)]
    branches = [torch.cuda.Stream() for _ in range(3)]
    preps = [{name: mvk.Prepared(layers[L].keys[name], B, ell) for (name, _, _, _) in stack.PROJECTIONS}
             for L in range(nl)]
    outs = [stack.LayerOutputs.allocate(B, ell) for _ in range(nl)]

    def check(tag):
        for L in range(nl):
            got = outs[L].as_dict()
            for name in ref[L]:
                for a, b in zip(ref[L][name], got[name]):
                    assert torch.equal(a, b), (tag, L, name)
        want = [1] * B
        want[3] = 0
        assert outs[1].accept["up"].tolist() == want

    def one_pass():
        stack.run_pass_overlapped(layers, inputs, preps, outs, main, preps_s, branches, tamper=tamper)

    with torch.cuda.stream(main):
        one_pass()
    torch.cuda.synchronize()
    check("eager")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=main):
        one_pass()
    for rep in range(3):
        for o in outs:
            for t in list(o.y.values()) + list(o.accept.values()) + list(o.yhat.values()):
                t.fill_(-1)
        torch.cuda.synchronize()
        with torch.cuda.stream(main):
            g.replay()
        torch.cuda.synchronize()
        check(f"replay {rep}")
    del g
