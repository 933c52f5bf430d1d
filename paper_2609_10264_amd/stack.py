"""A stack of decoder layers delegated with pvMVMD (Maverick's inference loop
restricted to its linear operations, Sec. 7.2).

Every layer has seven projections of a 4096-wide decoder block:
q, k, v, o (4096 x 4096), up, gate (11008 x 4096), down (4096 x 11008).
Per layer and batch of B query columns the client encodes four inputs
(q/k/v share one, up/gate share one), the server evaluates the seven products,
and the client verifies and decrypts the seven responses.  The nonlinear
operations between projections are outside this library: every input is a
fresh synthetic query.

Codes are shared per shape (one privacy code per input width n, one
verification code per output height m); P^T and Q are per matrix.  This module
only orchestrates calls of the C ABI (through the binding); all arithmetic runs
in the HIP kernels.

Schedules: run_layer (the one-call path: encode, server_eval, decode_verify,
one layer on one stream), prepare_layer + run_layer_prepared (the standard
mode with precomputation, Sec. 7: the masks and challenge vectors depend on
neither the queries nor the responses, so a preparation stream computes them
ahead and the online calls only add masks, evaluate and check), and
run_pass_overlapped (the same prepared work for a whole pass on several
streams, every data dependence of an inference pass kept as a stream edge).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import torch

from . import (Code, Key, PackedW, Prepared, client_prepare_group, client_prepare_multi, decode_verify, decode_verify_masked_group, encode,
               encode_masked, keygen, pack_weights, pack_weights_group, server_eval, server_eval_group)

# (name, m, n, input group)
PROJECTIONS = (
    ("q", 4096, 4096, "attn_in"),
    ("k", 4096, 4096, "attn_in"),
    ("v", 4096, 4096, "attn_in"),
    ("o", 4096, 4096, "attn_out"),
    ("up", 11008, 4096, "mlp_in"),
    ("gate", 11008, 4096, "mlp_in"),
    ("down", 4096, 11008, "mlp_out"),
)
INPUTS = ("attn_in", "attn_out", "mlp_in", "mlp_out")


@dataclass
class Layer:
    W: dict = field(default_factory=dict)       # name -> int8 m x n, or its PackedW
    keys: dict = field(default_factory=dict)    # name -> Key
    stacks: dict = field(default_factory=dict)  # input group -> (PackedW row stack, [names]) for shared inputs


def input_width(group: str) -> int:
    return next(n for (_, _, n, g) in PROJECTIONS if g == group)


def stage(group: str) -> list:
    """The projections fed by one input, in PROJECTIONS order."""
    return [name for (name, _, _, g) in PROJECTIONS if g == group]


def build_layer(weights: dict, cx_by_n: dict, cy_by_m: dict, stream=None, packed: bool = True) -> Layer:
    """Preprocess every projection of one layer (keygen on the device).  With
    `packed` the server keeps W in the packed matrix-core layout, and the
    projections that share an input (q, k, v; up, gate) as one row stack, so
    that one launch evaluates them together; layer.W[name] views its part."""
    layer = Layer()
    for name, m, n, _ in PROJECTIONS:
        W = weights[name]
        key = Key.allocate(m, n, cx_by_n[n], cy_by_m[m], device=W.device)
        keygen(key, W, stream=stream)
        layer.keys[name] = key
        if not packed:
            layer.W[name] = W
    if packed:
        for group in INPUTS:
            names = stage(group)
            if len(names) == 1:
                layer.W[names[0]] = pack_weights(weights[names[0]], stream=stream)
                continue
            st = pack_weights_group([weights[nm] for nm in names], stream=stream)
            nb = st.data.numel() // len(names)
            for g, nm in enumerate(names):
                m, n = weights[nm].shape
                layer.W[nm] = PackedW(st.data[g * nb:(g + 1) * nb], m, n)
            layer.stacks[group] = (st, names)
    return layer


def evaluate_stage(layer: Layer, group: str, Xhat: torch.Tensor, outs: dict | None = None, stream=None) -> dict:
    """The server's products for every projection fed by one input: one
    launch over the row stack where the layer keeps one, else one per
    projection.  Returns {name: Yhat}."""
    names = stage(group)
    if group in layer.stacks:
        st, _ = layer.stacks[group]
        res = server_eval_group(st, len(names), Xhat, outs=[outs[nm] for nm in names] if outs else None,
                                stream=stream)
        return dict(zip(names, res))
    return {nm: server_eval(layer.W[nm], Xhat, out=outs[nm] if outs else None, stream=stream) for nm in names}


def run_layer(layer: Layer, X: dict, ex: dict, ey: dict, tamper=None, stream=None):
    """One layer for a batch of query columns.

    X[group]: B x n plaintext queries; ex[group] = (idx, val) noise of that
    input (B x t_x); ey[name] = (idx, val) challenges (ell x t_y).
    tamper: optional callable(name, Yhat) applied to each response before
    verification (the test harness's dishonest server).
    Returns {name: (Y, accept, Xhat, Yhat, vL, vR)}.
    """
    Xhat = {}
    for group in INPUTS:
        # any projection fed by this input has the right privacy code
        name = next(p for (p, _, _, g) in PROJECTIONS if g == group)
        Xhat[group] = encode(layer.keys[name], X[group], ex[group][0], ex[group][1], stream=stream)
    out = {}
    Yhats = {}
    for group in INPUTS:
        Yhats.update(evaluate_stage(layer, group, Xhat[group], stream=stream))
    for name, m, n, group in PROJECTIONS:
        Yhat = Yhats[name]
        if tamper is not None:
            tamper(name, Yhat)
        ell, B = ey[name][0].shape[0], Yhat.shape[0]
        vL = torch.empty((ell, B), dtype=torch.int32, device=Yhat.device)
        vR = torch.empty_like(vL)
        Y, acc, _, _ = decode_verify(layer.keys[name], Xhat[group], Yhat, ex[group][0], ex[group][1],
                                     ey[name][0], ey[name][1], vL=vL, vR=vR, stream=stream)
        out[name] = (Y, acc, Xhat[group], Yhat, vL, vR)
    return out


def prepare_input(layer: Layer, group: str, ex: dict, ey: dict, preps: dict, flag: torch.Tensor | None = None,
                  stream=None) -> None:
    """Client preparation for the projections fed by one input: the input
    mask Gx e of its noise once, and per projection the output mask P e and
    the challenge vectors Gy e_q, e_q^T Q (one client_prepare_group launch).
    flag: an int32 device word set to 1 once every output is visible
    device-wide."""
    names = stage(group)
    B = ex[group][0].shape[0]
    for nm in names:
        if nm not in preps:
            preps[nm] = Prepared(layer.keys[nm], B, ey[nm][0].shape[0], device=ex[group][0].device)
    client_prepare_group([layer.keys[nm] for nm in names], ex[group][0], ex[group][1], [ey[nm] for nm in names],
                         outs=[preps[nm] for nm in names], done_flag=flag, stream=stream)


def prepare_layer(layer: Layer, ex: dict, ey: dict, flag: torch.Tensor | None, out: dict | None = None,
                  stream=None) -> dict:
    """Client preparation of one layer in one call (client_prepare_multi: the
    four inputs' masks and the seven projections' output masks and challenge
    vectors; one launch for the short syndromes and every row gather).
    flag: an int32 device word (or None) set to 1 once every output of the
    layer is visible device-wide, so one wait (the first masked encode of the
    layer's online part) covers the whole layer.  Returns {name: Prepared}."""
    preps = out if out is not None else {}
    keys, exs, eys, outs = [], [], [], []
    for name, _, _, group in PROJECTIONS:
        if name not in preps:
            preps[name] = Prepared(layer.keys[name], ex[group][0].shape[0], ey[name][0].shape[0],
                                   device=ex[group][0].device)
        keys.append(layer.keys[name])
        exs.append(ex[group])
        eys.append(ey[name])
        outs.append(preps[name])
    done = [flag] + [None] * (len(keys) - 1) if flag is not None else None
    client_prepare_multi(keys, exs, eys, outs=outs, done_flags=done, stream=stream)
    return preps


def check_stage(layer: Layer, group: str, Xhat: torch.Tensor, Yhats: dict, preps: dict, out: dict | None = None,
                stream=None) -> dict:
    """The client's Verify + Decrypt for the projections fed by one input (one
    decode_verify_masked_group launch where the problem allows).  out:
    {name: (Y, accept, vL, vR)} preallocated, or None.  Returns the same."""
    names = stage(group)
    B = Xhat.shape[0]
    dev_ = Xhat.device
    res = {}
    for nm in names:
        if out is not None:
            res[nm] = out[nm]
        else:
            ell = preps[nm].ell
            m = layer.keys[nm].m
            res[nm] = (torch.empty((B, m), dtype=torch.int32, device=dev_),
                       torch.empty((B,), dtype=torch.int32, device=dev_),
                       torch.empty((ell, B), dtype=torch.int32, device=dev_),
                       torch.empty((ell, B), dtype=torch.int32, device=dev_))
    decode_verify_masked_group([layer.keys[nm] for nm in names], Xhat, [Yhats[nm] for nm in names],
                               [preps[nm] for nm in names], Ys=[res[nm][0] for nm in names],
                               vLs=[res[nm][2] for nm in names], vRs=[res[nm][3] for nm in names],
                               accepts=[res[nm][1] for nm in names], stream=stream)
    return res


def run_layer_prepared(layer: Layer, X: dict, preps: dict, ready_flag: torch.Tensor | None = None,
                       timeout_us: int = 200000, timed_out: torch.Tensor | None = None, tamper=None, stream=None):
    """The online part of a layer with prepared masks, input by input as in
    inference: x^ = x + Gx e, the server's products for that input (one
    grouped launch for q, k, v and for up, gate), and their checks
    (decode_verify_masked_group).  ready_flag: one device word (the layer's
    last preparation flag, waited for by the first masked encode) or a list of
    four, one per input (each masked encode waits for its own).  Every wait
    clears its flag.  Same outputs as run_layer with the same noise and
    challenges."""
    out = {}
    for i, group in enumerate(INPUTS):
        names = stage(group)
        wait = ready_flag[i] if isinstance(ready_flag, (list, tuple)) else (ready_flag if i == 0 else None)
        xh = encode_masked(layer.keys[names[0]], X[group], preps[names[0]], ready_flag=wait, timeout_us=timeout_us,
                           timed_out=timed_out, stream=stream)
        Yhats = evaluate_stage(layer, group, xh, stream=stream)
        if tamper is not None:
            for nm in names:
                tamper(nm, Yhats[nm])
        checked = check_stage(layer, group, xh, Yhats, preps, stream=stream)
        for nm in names:
            Y, acc, vL, vR = checked[nm]
            out[nm] = (Y, acc, xh, Yhats[nm], vL, vR)
    return out


@dataclass
class LayerOutputs:
    """Preallocated outputs of one layer for run_pass_overlapped: X^ per input,
    and per projection Y^, Y, v_L, v_R and the accept bits."""
    xhat: dict = field(default_factory=dict)
    yhat: dict = field(default_factory=dict)
    y: dict = field(default_factory=dict)
    vl: dict = field(default_factory=dict)
    vr: dict = field(default_factory=dict)
    accept: dict = field(default_factory=dict)

    @classmethod
    def allocate(cls, B: int, ell: int, device="cuda") -> "LayerOutputs":
        o = cls()
        i32 = dict(dtype=torch.int32, device=device)
        for group in INPUTS:
            o.xhat[group] = torch.empty((B, input_width(group)), **i32)
        for name, m, n, _ in PROJECTIONS:
            o.yhat[name] = torch.empty((B, m), **i32)
            o.y[name] = torch.empty((B, m), **i32)
            o.vl[name] = torch.empty((ell, B), **i32)
            o.vr[name] = torch.empty((ell, B), **i32)
            o.accept[name] = torch.empty((B,), **i32)
        return o

    def as_dict(self) -> dict:
        """{name: (Y, accept, Xhat, Yhat, vL, vR)}, as run_layer returns."""
        return {name: (self.y[name], self.accept[name], self.xhat[group], self.yhat[name], self.vl[name],
                       self.vr[name]) for name, _, _, group in PROJECTIONS}


def run_pass_overlapped(layers: list, inputs: list, preps: list, outs: list, main, prep_streams: list,
                        branch_streams: list = (), tamper=None):
    """One pass over every layer, issued on several streams so that work
    without a data dependence runs side by side; captured on `main`, the
    streams fork from it and join it again, so a HIP graph of the pass keeps
    every dependence below as an edge.

    Dependences kept (the rest runs concurrently):
      * the client's preparation of a projection (client_prepare: masks and
        challenge vectors, independent of queries and responses, Sec. 7)
        runs on the preparation streams, one layer ahead of the online part;
        a layer's online part waits for its preparation;
      * per layer the inputs follow one another as in inference: q, k, v
        share one input, o's input comes after the q, k, v outputs, up and
        gate share the next, down's comes last; each input's masked encode
        waits for every verification of the previous stage;
      * within a stage the server's products (one launch over the row stack
        of the projections that share the input), then their checks (one
        grouped decode/verify launch), on the main stream.
    inputs[L] = (X, ex, ey) as for run_layer; preps[L]: {name: Prepared};
    outs[L]: LayerOutputs; tamper: optional callable(L, name, Yhat) on the
    branch stream between the product and its check."""
    every = list(prep_streams) + list(branch_streams)
    for s in every:
        s.wait_stream(main)

    def prepare(L):
        _, ex, ey = inputs[L]
        if len(prep_streams) == 1:  # the whole layer in one call
            with torch.cuda.stream(prep_streams[0]):
                prepare_layer(layers[L], ex, ey, None, out=preps[L], stream=prep_streams[0])
        else:
            for k, group in enumerate(INPUTS):
                s = prep_streams[k % len(prep_streams)]
                with torch.cuda.stream(s):
                    prepare_input(layers[L], group, ex, ey, preps[L], stream=s)
        return [s.record_event() for s in prep_streams]

    ready = {0: prepare(0)} if layers else {}
    for L, layer in enumerate(layers):
        if L + 1 < len(layers):
            ready[L + 1] = prepare(L + 1)
        for e in ready.pop(L):
            main.wait_event(e)
        X = inputs[L][0]
        o = outs[L]
        for group in INPUTS:
            names = stage(group)
            with torch.cuda.stream(main):
                encode_masked(layer.keys[names[0]], X[group], preps[L][names[0]], out=o.xhat[group], stream=main)
                evaluate_stage(layer, group, o.xhat[group], outs=o.yhat, stream=main)
            with torch.cuda.stream(main):
                if tamper is not None:
                    for name in names:
                        tamper(L, name, o.yhat[name])
                check_stage(layer, group, o.xhat[group], o.yhat, preps[L],
                            out={nm: (o.y[nm], o.accept[nm], o.vl[nm], o.vr[nm]) for nm in names}, stream=main)
    for s in every:
        main.wait_stream(s)


def codes_for(make_code) -> tuple[dict, dict]:
    """Shared codes: privacy code per input width, verification code per output height."""
    ns = sorted({n for (_, _, n, _) in PROJECTIONS})
    ms = sorted({m for (_, m, _, _) in PROJECTIONS})
    return {n: make_code("x", n) for n in ns}, {m: make_code("y", m) for m in ms}


def macs_per_layer(B: int) -> int:
    return sum(m * n for (_, m, n, _) in PROJECTIONS) * B


__all__ = ["PROJECTIONS", "INPUTS", "Layer", "LayerOutputs", "build_layer", "evaluate_stage", "check_stage",
           "run_layer", "prepare_input", "prepare_layer", "run_layer_prepared", "run_pass_overlapped", "codes_for",
           "input_width", "stage", "macs_per_layer", "Code"]
