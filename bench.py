"""Benchmark of the pvMVMD hot path on one MI355X.

One step = one pass of the whole hot path over one batch of query columns:
    encode (Encrypt: x^ = x + Gx e_x)  ->  server_eval (y^ = W x^ mod p)
    ->  decode_verify (Verify with ell sparse challenges + Decrypt)
on the 4096 x 4096 attention-projection workload (one query column, r = 3,
t_x = 64, t_y = 31, ell = 2, p = 2^31 - 1, W int8-valued).  All inputs are
resident in HBM before the timed region.  A pool of distinct weight matrices
(each with its own preprocessed P^T and Q) is cycled so that consecutive steps
never find W in the 256 MB last-level cache.

Printed JSON line:
  value       modMAC/s of the whole step (m*n*B per step / step time)
  roofline    server_eval kernel: algorithmic bytes (m*n + 4*n*B + 4*m*B) per
              launch / mean launch duration (HIP events around each launch on
              the launch stream), against 8 TB/s HBM
  cpu_baseline the CPU oracle (single-threaded plain C) on a bounded sample of
              the same steps, on this host
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "server_eval mod-MACs/s + achieved HBM GB/s (fraction of peak), 1×MI355X"
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="attn4096")
    ap.add_argument("--pool", type=int, default=0, help="distinct W matrices cycled (0: enough for 2x the LLC)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="time budget of the CPU oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--seed", type=int, default=2609)
    ap.add_argument("--path", default="auto", choices=["auto", "valu", "mfma"], help="server_eval kernel family")
    ap.add_argument("--m", type=int, default=0, help="override the workload's row count (server-only)")
    ap.add_argument("--n", type=int, default=0, help="override the workload's column count (server-only)")
    ap.add_argument("--B", type=int, default=0, help="override the workload's query count (server-only)")
    ap.add_argument("--server-only", action="store_true",
                    help="time server_eval alone (no client steps) on the chosen workload")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; multi-GPU runs are not supported",
                          "n_gpus": args.gpus}), flush=True)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2609_10264_amd as mvk
    import synth

    torch.cuda.set_device(0)
    cfg = dict(synth.CONFIGS[args.config])
    if args.server_only:
        for key in ("m", "n", "B"):
            if getattr(args, key):
                cfg[key] = getattr(args, key)
    m, n, B, r, tx, ty, ell = (cfg[k] for k in ("m", "n", "B", "r", "tx", "ty", "ell"))
    cid = cfg["cid"]
    w_bytes = m * n
    pool = args.pool or max(2, -(-2 * 256 * 2**20 // w_bytes))
    total_steps = args.warmup + args.steps
    dev = torch.device("cuda")

    def d(a):
        a = np.ascontiguousarray(a)
        return torch.from_numpy(a.astype(np.int32) if a.dtype != np.int8 else a).to(dev)

    if args.server_only:
        return server_only(args, cfg, pool, total_steps, dev)

    # ---- setup (untimed) ---------------------------------------------------
    cx_h = synth.raa_code(synth.seed_for(cid, synth.PURPOSE_CX), n, r)
    cy_h = synth.raa_code(synth.seed_for(cid, synth.PURPOSE_CY), m, r)

    def code(c):
        return mvk.Code(c["k"], c["r"], d(c["pi1"]), d(c["pi2"]), d(c["v1"]), d(c["v2"]))

    cx, cy = code(cx_h), code(cy_h)
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed)
    Ws, keys = [], []
    for j in range(pool):
        Wj = torch.randint(-127, 128, (m, n), generator=gen, device=dev, dtype=torch.int8)
        kj = mvk.Key.allocate(m, n, cx, cy)
        mvk.keygen(kj, Wj)
        Ws.append(Wj)
        keys.append(kj)
    X = torch.randint(0, mvk.P, (total_steps, B, n), generator=gen, device=dev, dtype=torch.int32)
    exi, exv = synth.sparse(synth.seed_for(cid, synth.PURPOSE_NOISE, 7), total_steps * B, cx.N, tx)
    eyi, eyv = synth.sparse(synth.seed_for(cid, synth.PURPOSE_CHAL, 7), total_steps * ell, cy.N, ty)
    EXI, EXV = d(exi).view(total_steps, B, tx), d(exv).view(total_steps, B, tx)
    EYI, EYV = d(eyi).view(total_steps, ell, ty), d(eyv).view(total_steps, ell, ty)
    Xh = torch.empty((B, n), dtype=torch.int32, device=dev)
    Yh = torch.empty((B, m), dtype=torch.int32, device=dev)
    Y = torch.empty((B, m), dtype=torch.int32, device=dev)
    ACC = torch.zeros((total_steps, B), dtype=torch.int32, device=dev)
    torch.cuda.synchronize()

    ev0 = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ev1 = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]

    def step(i, timed_idx=None):
        j = i % pool
        mvk.encode(keys[j], X[i], EXI[i], EXV[i], out=Xh)
        if timed_idx is not None:
            ev0[timed_idx].record()
        mvk.server_eval(Ws[j], Xh, out=Yh, path=args.path)
        if timed_idx is not None:
            ev1[timed_idx].record()
        mvk.decode_verify(keys[j], Xh, Yh, EXI[i], EXV[i], EYI[i], EYV[i], Y=Y, accept=ACC[i])

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(args.warmup + s, s)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    elapsed = t1 - t0
    se_ms = [a.elapsed_time(b) for a, b in zip(ev0, ev1)]
    accepted = bool((ACC == 1).all().item())

    macs = m * n * B
    ms_per_step = 1e3 * elapsed / args.steps
    se_mean_s = 1e-3 * float(np.mean(se_ms))
    alg_bytes = m * n + 4 * n * B + 4 * m * B
    achieved = alg_bytes / se_mean_s / 1e9

    out = {
        "metric": METRIC,
        "value": macs * args.steps / elapsed,
        "unit": "modMAC/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i8xi8->i32 limb dot products, mod 2^31-1",
        "data": "synthetic",
        "config": {"workload": f"{args.config}: W {m}x{n} int8-valued in F_p (p=2^31-1), B={B} query column(s), "
                               f"RAA r={r}, t_x={tx}, t_y={ty}, ell={ell}; step = encode+server_eval+decode_verify",
                   "global_batch": B, "w_pool": pool},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "kernel": f"server_eval ({args.path})", "alg_bytes_per_launch": alg_bytes,
                     "mean_launch_us": 1e6 * se_mean_s, "median_launch_us": 1e3 * float(np.median(se_ms))},
        "server_eval": {"modmac_per_s": macs / se_mean_s, "gb_per_s": achieved},
        "all_accepted": accepted,
    }

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args, cfg, cx_h, cy_h)
    print(json.dumps(out), flush=True)
    if not accepted:
        sys.exit(1)


def server_only(args, cfg, pool, total_steps, dev):
    """server_eval alone over a rotated pool of W; events around every launch."""
    import numpy as np
    import torch

    import paper_2609_10264_amd as mvk

    m, n, B = cfg["m"], cfg["n"], cfg["B"]
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed)
    Ws = [torch.randint(-127, 128, (m, n), generator=gen, device=dev, dtype=torch.int8) for _ in range(pool)]
    X = torch.randint(0, mvk.P, (pool, B, n), generator=gen, device=dev, dtype=torch.int32)
    Y = torch.empty((B, m), dtype=torch.int32, device=dev)
    for i in range(args.warmup):
        mvk.server_eval(Ws[i % pool], X[i % pool], out=Y, path=args.path)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        ev[i][0].record()
        mvk.server_eval(Ws[i % pool], X[i % pool], out=Y, path=args.path)
        ev[i][1].record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms = np.array([a.elapsed_time(b) for a, b in ev])
    mean_s = 1e-3 * float(ms.mean())
    alg_bytes = m * n + 4 * n * B + 4 * m * B
    macs = m * n * B
    out = {"metric": METRIC, "value": macs / mean_s, "unit": "modMAC/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": 1e3 * elapsed / args.steps, "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "i8xi8->i32 limb dot products, mod 2^31-1",
           "data": "synthetic",
           "config": {"workload": f"{args.config}: server_eval only, W {m}x{n} int8-valued, B={B}",
                      "global_batch": B, "w_pool": pool},
           "roofline": {"bound": "hbm", "achieved": alg_bytes / mean_s / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": alg_bytes / mean_s / 1e9 / HBM_PEAK_GBS, "traffic": None,
                        "kernel": f"server_eval ({args.path})", "alg_bytes_per_launch": alg_bytes,
                        "mean_launch_us": 1e6 * mean_s, "median_launch_us": 1e3 * float(np.median(ms))},
           "mfma_int8_tops": 2 * 4 * macs / mean_s / 1e12}
    print(json.dumps(out), flush=True)


def cpu_baseline(args, cfg, cx_h, cy_h):
    """Oracle step (encode, server_eval, verify, decode) timed on a bounded sample."""
    import numpy as np

    import oracle
    import synth

    m, n, B, tx, ty, ell = (cfg[k] for k in ("m", "n", "B", "tx", "ty", "ell"))
    cid = cfg["cid"]
    W = synth.weights(synth.seed_for(cid, synth.PURPOSE_W, 5), m, n)
    PT, Q = oracle.keygen(W, cx_h, cy_h)  # preprocessing, untimed
    steps = 0
    el = 0.0
    while True:
        X = synth.field_uniform(synth.seed_for(cid, synth.PURPOSE_X, 100 + steps), (B, n))
        exi, exv = synth.sparse(synth.seed_for(cid, synth.PURPOSE_NOISE, 100 + steps), B, cx_h["N"], tx)
        eyi, eyv = synth.sparse(synth.seed_for(cid, synth.PURPOSE_CHAL, 100 + steps), ell, cy_h["N"], ty)
        t0 = time.perf_counter()
        Xh = oracle.encode(cx_h, X, exi, exv)
        Yh = oracle.server_eval(W, Xh)
        acc, _, _ = oracle.verify(cy_h, Q, Xh, Yh, eyi, eyv)
        oracle.decode(PT, Yh, exi, exv)
        el += time.perf_counter() - t0
        assert acc.all()
        steps += 1
        if el >= args.cpu_seconds or steps >= 10000:
            break
    return {"value": m * n * B * steps / el, "unit": "modMAC/s", "cores": 1, "kind": "oracle",
            "sample": f"{steps} full steps (encode+server_eval+verify+decode) of the same workload, one W, "
                      f"{el:.1f} s of oracle time (input drawing excluded); single-threaded C, '%' per field op"}


if __name__ == "__main__":
    main()
