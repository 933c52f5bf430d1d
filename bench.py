"""Benchmark of the pvMVMD hot path on one MI355X.

One step = one pass of the whole hot path over one batch of query columns:
    encode (Encrypt: x^ = x + Gx e_x)  ->  server_eval (y^ = W x^ mod p)
    ->  decode_verify (Verify with ell sparse challenges + Decrypt)
on the 4096 x 4096 attention-projection workload (one query column, r = 3,
t_x = 64, t_y = 31, ell = 2, p = 2^31 - 1, W int8-valued).  All inputs are
resident in HBM before the timed region.  A pool of distinct weight matrices
(each with its own preprocessed P^T and Q) is cycled so that consecutive steps
never find W in the 256 MB last-level cache.

Two schedules of the same work (--mode):
  pipelined   the paper's standard mode with pipelining (Sec. 7): the work that
              depends on neither the query nor the response (masks Gx e_x and
              P e_x, challenge vectors Gy e_q and e_q^T Q; client_prepare) runs
              on a preparation stream ahead of the online stream
              (encode_masked -> server_eval -> decode_verify_masked); stream
              flags order each step after its own preparation.  Both streams
              replay one HIP graph each, concurrently.
  serial      every step's calls back to back on one stream (encode ->
              server_eval -> decode_verify), one HIP graph.
Every timed step does all of its work inside the timed region in both.

Printed JSON line:
  value       modMAC/s of the whole step (m*n*B per step / step time), in the
              chosen mode; the other mode's step time is printed beside it
  roofline    server_eval kernel: algorithmic bytes (m*n + 4*n*B + 4*m*B) per
              launch / mean launch duration (HIP events around each launch on
              the launch stream), against 8 TB/s HBM
              read_floor: a pure streaming read (mvk_stream_read) of the same
              buffers timed the same way; frac = read time / server_eval time
  server_eval_large  the same single-query kernel at 16384 x 16384 (268 MB of
              W per launch), where streaming W dominates the launch
  server_eval_batched  the 64-query kernel at 28672 x 8192 against the int8
              matrix-core peak (4 digit-plane multiply-adds per mod-MAC)
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
MFMA_INT8_PEAK_OPS = 5.0e15  # MI355X dense int8 matrix-core peak
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "server_eval_attn4096_traffic.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2609_10264_amd", "csrc", "server_eval.hip")


def kernel_src_sha256() -> str:
    import hashlib
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(config: str, weights: str):
    """HBM bytes per server_eval launch from the committed counter runs, if they
    were taken on the current kernel source, this workload and weight layout;
    else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
        sha = kernel_src_sha256()
    except OSError:
        return None
    if rec.get("kernel_src_sha256") != sha or rec.get("config") != config or rec.get("weights") != weights:
        return None
    return rec.get("traffic_bytes_per_launch")


def write_traffic(fetch_csv: str, write_csv: str, config: str, weights: str, copy_mib: int, kernel_match: str):
    """Traffic record from two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE; KiB
    per dispatch) of `bench.py --calib-copy-mib copy_mib`: the server_eval
    kernel's medians, each scaled by what the same counter reads for the
    copy_mib MiB device copy (which reads and writes copy_mib MiB)."""
    import csv
    import statistics

    def per_kernel(path, counter):
        vals, copies = [], []
        with open(path) as f:
            for row in csv.DictReader(f):
                if row["Counter_Name"] != counter:
                    continue
                v = float(row["Counter_Value"])
                if kernel_match in row["Kernel_Name"]:
                    vals.append(v)
                elif "copyBuffer" in row["Kernel_Name"]:
                    copies.append(v)
        if not vals or not copies:
            raise SystemExit(f"{path}: no {counter} rows for {kernel_match!r} or the copy kernel")
        return statistics.median(vals), len(vals), max(copies)

    f_med, f_n, f_copy = per_kernel(fetch_csv, "FETCH_SIZE")
    w_med, w_n, w_copy = per_kernel(write_csv, "WRITE_SIZE")
    ref_kib = copy_mib * 1024.0
    fs, ws = ref_kib / f_copy, ref_kib / w_copy
    rec = {"kernel": kernel_match, "config": config, "weights": weights, "kernel_src_sha256": kernel_src_sha256(),
           "fetch_size_kib_per_dispatch": f_med, "write_size_kib_per_dispatch": w_med, "dispatches": [f_n, w_n],
           "copy_reference_mib": copy_mib, "copy_fetch_size_kib": f_copy, "copy_write_size_kib": w_copy,
           "fetch_scale": fs, "write_scale": ws,
           "traffic_bytes_per_launch": int(round((f_med * fs + w_med * ws) * 1024))}
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))


def calib_copy(mib: int):
    import torch
    src = torch.ones(mib * 2**20, dtype=torch.int8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()


def warm(replay, seconds):
    """Untimed replays until `seconds` have passed: the GPU's clocks ramp up
    under sustained load, and a timed replay right after setup reads up to
    ~15% slow."""
    import torch

    t_end = time.perf_counter() + seconds
    while True:
        replay()
        torch.cuda.synchronize()
        if time.perf_counter() >= t_end:
            return


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="attn4096",
                    help="attn4096 (default), mlp_up_11008x4096, mlp_large_28672x8192, tiny, stack32 or paper_eval "
                         "(the Sec. 7.1 BabyBear sweep; --n picks one size)")
    ap.add_argument("--pool", type=int, default=0, help="distinct W matrices cycled (0: enough for 2x the LLC)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="time budget of the CPU oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-large", action="store_true",
                    help="skip the 16384 x 16384 single-query and 28672 x 8192 64-query server_eval "
                         "measurements of the default line")
    ap.add_argument("--eager", action="store_true", help="launch the timed steps one by one instead of a HIP graph")
    ap.add_argument("--chains", type=int, default=1,
                    help="serial schedule: independent query chains run side by side (step i belongs to chain "
                         "i mod chains)")
    ap.add_argument("--mode", default="pipelined", choices=["pipelined", "serial"],
                    help="schedule of the timed steps whose time gives `value` (both are measured)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after timing, copy this many MiB device-to-device (reference kernel for HBM counters)")
    ap.add_argument("--seed", type=int, default=2609)
    ap.add_argument("--warm-seconds", type=float, default=0.3,
                    help="untimed replays of each timed graph before its timed replay")
    ap.add_argument("--path", default="auto", choices=["auto", "valu", "mfma"], help="server_eval kernel family")
    ap.add_argument("--write-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the server_eval traffic record from two rocprofv3 --pmc counter files and exit")
    ap.add_argument("--traffic-kernel", default="server_eval_mfma_small<1, 8, 8, true, 2>",
                    help="kernel name fragment the traffic record is taken for")
    ap.add_argument("--weights", default="packed", choices=["packed", "rowmajor"],
                    help="server weight layout: packed once into matrix-core operand order (untimed, like "
                         "keygen), or row-major as given")
    ap.add_argument("--m", type=int, default=0, help="override the workload's row count (server-only)")
    ap.add_argument("--n", type=int, default=0, help="override the workload's column count (server-only)")
    ap.add_argument("--B", type=int, default=0, help="override the workload's query count (server-only)")
    ap.add_argument("--server-only", action="store_true",
                    help="time server_eval alone (no client steps) on the chosen workload")
    ap.add_argument("--batch-verify", type=int, default=0, metavar="B",
                    help="time batch verification (Protocol Batch-vMVMD) of B claims of the workload's shape "
                         "against B one-claim verifications, and exit")
    return ap.parse_args()


def main():
    args = parse()
    if args.write_traffic:
        return write_traffic(args.write_traffic[0], args.write_traffic[1], args.config, args.weights,
                             args.calib_copy_mib or 256, args.traffic_kernel)
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; multi-GPU runs are not supported",
                          "n_gpus": args.gpus}), flush=True)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2609_10264_amd as mvk
    import synth

    torch.cuda.set_device(0)
    if args.config == "stack32":
        return stack_bench(args)
    if args.batch_verify:
        return batch_verify_bench(args)
    if args.config == "paper_eval":
        return paper_eval_bench(args)
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
        Ws.append(mvk.pack_weights(Wj) if args.weights == "packed" else Wj)
        keys.append(kj)
    X = torch.randint(0, mvk.P, (total_steps, B, n), generator=gen, device=dev, dtype=torch.int32)
    exi, exv = synth.sparse(synth.seed_for(cid, synth.PURPOSE_NOISE, 7), total_steps * B, cx.N, tx)
    eyi, eyv = synth.sparse(synth.seed_for(cid, synth.PURPOSE_CHAL, 7), total_steps * ell, cy.N, ty)
    EXI, EXV = d(exi).view(total_steps, B, tx), d(exv).view(total_steps, B, tx)
    EYI, EYV = d(eyi).view(total_steps, ell, ty), d(eyv).view(total_steps, ell, ty)
    C = max(1, args.chains)
    if args.warmup < C:
        raise SystemExit("--warmup must be at least --chains (each chain warms its own stream)")
    # per chain: its own stream, its own output buffers
    streams = [torch.cuda.Stream() for _ in range(C)]
    Xh = [torch.empty((B, n), dtype=torch.int32, device=dev) for _ in range(C)]
    Yh = [torch.empty((B, m), dtype=torch.int32, device=dev) for _ in range(C)]
    Y = [torch.empty((B, m), dtype=torch.int32, device=dev) for _ in range(C)]
    ACC = torch.zeros((total_steps, B), dtype=torch.int32, device=dev)
    torch.cuda.synchronize()

    def step(i):
        """Step i on chain i % C (launched on the current stream = that chain's)."""
        j, c = i % pool, i % C
        mvk.encode(keys[j], X[i], EXI[i], EXV[i], out=Xh[c])
        mvk.server_eval(Ws[j], Xh[c], out=Yh[c], path=args.path)
        mvk.decode_verify(keys[j], Xh[c], Yh[c], EXI[i], EXV[i], EYI[i], EYV[i], Y=Y[c], accept=ACC[i])

    # warm-up on the launch streams (also sizes the library's per-stream workspaces)
    for i in range(args.warmup):
        with torch.cuda.stream(streams[i % C]):
            step(i)
    torch.cuda.synchronize()
    timed = [[args.warmup + k for k in range(args.steps) if (args.warmup + k) % C == c] for c in range(C)]

    if args.eager:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(args.steps):
            i = args.warmup + k
            with torch.cuda.stream(streams[i % C]):
                step(i)
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
    else:
        # Each chain's timed steps are captured once as a HIP graph on its own
        # stream and replayed: identical kernels and inputs, without per-launch
        # host gaps.  Steps of one chain run in order; with C > 1 the chains
        # (independent queries) run side by side.
        graphs = []
        for c in range(C):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=streams[c]):
                for i in timed[c]:
                    step(i)
            graphs.append(g)

        def replay_all():
            for c in range(C):
                with torch.cuda.stream(streams[c]):
                    graphs[c].replay()

        warm(replay_all, args.warm_seconds)  # untimed replays
        ACC.zero_()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        replay_all()
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
    accepted = bool((ACC[args.warmup:] == 1).all().item())
    # The buffers hold the last timed step of every chain; recompute those
    # steps eagerly and compare.
    last = [(Xh[c].clone(), Yh[c].clone(), Y[c].clone()) for c in range(C) if timed[c]]
    for c in range(C):
        if timed[c]:
            with torch.cuda.stream(streams[c]):
                step(timed[c][-1])
    torch.cuda.synchronize()
    now = [(Xh[c], Yh[c], Y[c]) for c in range(C) if timed[c]]
    replay_matches_eager = all(bool(torch.equal(a, b)) for la, lb in zip(last, now) for a, b in zip(la, lb))
    elapsed_serial, accepted_serial = elapsed, accepted

    # ---- pipelined standard mode -------------------------------------------
    # Step i's preparation (client_prepare, which sets step i's flag when its
    # outputs are visible) on the preparation stream; its online part
    # (encode_masked, which first waits for that flag, then server_eval and
    # decode_verify_masked) on the online stream.  One graph per stream over
    # all timed steps; the two replays run side by side.
    preps = [mvk.Prepared(keys[i % pool], B, ell) for i in range(total_steps)]
    flags = torch.zeros(total_steps, dtype=torch.int32, device=dev)
    late = torch.zeros((), dtype=torch.int32, device=dev)
    ACC2 = torch.zeros((total_steps, B), dtype=torch.int32, device=dev)
    s_prep, s_on = torch.cuda.Stream(), torch.cuda.Stream()
    pXh = torch.empty((B, n), dtype=torch.int32, device=dev)
    pYh = torch.empty((B, m), dtype=torch.int32, device=dev)
    pY = torch.empty((B, m), dtype=torch.int32, device=dev)

    def prepare(i):
        j = i % pool
        mvk.client_prepare(keys[j], EXI[i], EXV[i], EYI[i], EYV[i], out=preps[i], done_flag=flags[i])

    def online(i):
        j = i % pool
        mvk.encode_masked(keys[j], X[i], preps[i], out=pXh, ready_flag=flags[i], timeout_us=50_000, timed_out=late)
        mvk.server_eval(Ws[j], pXh, out=pYh, path=args.path)
        mvk.decode_verify_masked(keys[j], pXh, pYh, preps[i], Y=pY, accept=ACC2[i])

    for i in range(args.warmup):  # also sizes the library's per-stream workspaces
        with torch.cuda.stream(s_prep):
            prepare(i)
    for i in range(args.warmup):
        with torch.cuda.stream(s_on):
            online(i)
    torch.cuda.synchronize()
    steps_t = list(range(args.warmup, total_steps))
    g_prep, g_on = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_prep, stream=s_prep):
        for i in steps_t:
            prepare(i)
    with torch.cuda.graph(g_on, stream=s_on):
        for i in steps_t:
            online(i)

    def replay_pipelined():
        # The preparation graph is submitted first: HIP multiplexes streams onto
        # a few hardware queues, and a wait queued ahead of its signal on a
        # shared queue would only end at its time-out.
        with torch.cuda.stream(s_prep):
            g_prep.replay()
        with torch.cuda.stream(s_on):
            g_on.replay()

    warm(replay_pipelined, args.warm_seconds)  # untimed replays
    ACC2.zero_()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    replay_pipelined()
    torch.cuda.synchronize()
    elapsed_pipe = time.perf_counter() - t0
    accepted_pipe = bool((ACC2[args.warmup:] == 1).all().item()) and int(late.item()) == 0
    # the last timed step again through the one-call path: same Xhat, Yhat, Y
    i_last = steps_t[-1]
    got = (pXh.clone(), pYh.clone(), pY.clone())
    with torch.cuda.stream(s_on):
        rXh = mvk.encode(keys[i_last % pool], X[i_last], EXI[i_last], EXV[i_last])
        rYh = mvk.server_eval(Ws[i_last % pool], rXh, path=args.path)
        rY, _, _, _ = mvk.decode_verify(keys[i_last % pool], rXh, rYh, EXI[i_last], EXV[i_last], EYI[i_last],
                                        EYV[i_last])
    torch.cuda.synchronize()
    pipe_matches = all(bool(torch.equal(a, b)) for a, b in zip(got, (rXh, rYh, rY)))
    if args.mode == "pipelined":
        elapsed, accepted = elapsed_pipe, accepted_pipe
    s = streams[0]
    Yh = Yh[0]

    # server_eval alone, same W pool and masked queries, captured back to back;
    # HIP events on the launch stream bracket the replay.
    reps = args.steps
    Xs = torch.randint(0, mvk.P, (pool, B, n), generator=gen, device=dev, dtype=torch.int32)
    ge = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        for j in range(pool):
            mvk.server_eval(Ws[j], Xs[j], out=Yh, path=args.path)
    torch.cuda.synchronize()
    with torch.cuda.graph(ge, stream=s):
        for k in range(reps):
            mvk.server_eval(Ws[k % pool], Xs[k % pool], out=Yh, path=args.path)
    def replay_ge():
        with torch.cuda.stream(s):
            ge.replay()

    warm(replay_ge, args.warm_seconds)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(s):
        e0.record()
        ge.replay()
        e1.record()
    torch.cuda.synchronize()
    se_mean_s = 1e-3 * e0.elapsed_time(e1) / reps
    read_s = read_floor([w.data if isinstance(w, mvk.PackedW) else w for w in Ws], reps, args)
    large = None if args.no_large else server_eval_large(args, gen, dev)
    batched = None if args.no_large else server_eval_batched(args, gen, dev)

    macs = m * n * B
    ms_per_step = 1e3 * elapsed / args.steps
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
                   "global_batch": B, "w_pool": pool, "launch": "eager" if args.eager else "hip_graph",
                   "mode": args.mode, "chains": C if args.mode == "serial" else 1, "weights": args.weights},
        "ms_per_step_pipelined": 1e3 * elapsed_pipe / args.steps,
        "ms_per_step_serial": 1e3 * elapsed_serial / args.steps,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": measured_traffic(args.config, args.weights),
                     "kernel": f"server_eval ({args.path})", "alg_bytes_per_launch": alg_bytes,
                     "mean_launch_us": 1e6 * se_mean_s,
                     "read_floor": {"mean_launch_us": 1e6 * read_s, "gbps": alg_bytes / read_s / 1e9,
                                    "frac": read_s / se_mean_s}},
        "server_eval": {"modmac_per_s": macs / se_mean_s, "gb_per_s": achieved},
        "server_eval_large": large,
        "server_eval_batched": batched,
        "all_accepted": accepted_serial and accepted_pipe,
        "replay_matches_eager": replay_matches_eager,
        "pipelined_matches_one_call_path": pipe_matches,
    }

    if args.calib_copy_mib:
        calib_copy(args.calib_copy_mib)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args, cfg, cx_h, cy_h)
    print(json.dumps(out), flush=True)
    if not (accepted_serial and accepted_pipe and replay_matches_eager and pipe_matches):
        sys.exit(1)


def read_floor(bufs, reps, args):
    """Seconds per launch of a pure streaming read (mvk_stream_read) of the same
    buffers, back to back over the pool as the server_eval launches are: the
    measured read floor for that many bytes."""
    import torch

    import paper_2609_10264_amd as mvk

    s = torch.cuda.Stream()
    sink = torch.empty((mvk._lib.MVK_STREAM_READ_BLOCKS,), dtype=torch.int32, device=bufs[0].device)
    with torch.cuda.stream(s):
        for b in bufs:
            mvk.stream_read(b, sink, stream=s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for k in range(reps):
            mvk.stream_read(bufs[k % len(bufs)], sink, stream=s)

    def replay():
        with torch.cuda.stream(s):
            g.replay()

    warm(replay, args.warm_seconds)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(s):
        e0.record()
        g.replay()
        e1.record()
    torch.cuda.synchronize()
    return 1e-3 * e0.elapsed_time(e1) / reps


def server_eval_large(args, gen, dev, m=16384, n=16384, pool=2, reps=40):
    """The same single-query kernel where W streaming dominates: 16384 x 16384
    (268 MB of packed W per launch, a pool of two), HIP events around a graph of
    back-to-back launches on the launch stream."""
    import torch

    import paper_2609_10264_amd as mvk

    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        Ws = []
        for _ in range(pool):
            W = torch.randint(-127, 128, (m, n), generator=gen, device=dev, dtype=torch.int8)
            Ws.append(mvk.pack_weights(W, stream=s))
            del W
        X = torch.randint(0, mvk.P, (pool, 1, n), generator=gen, device=dev, dtype=torch.int32)
        Y = torch.empty((1, m), dtype=torch.int32, device=dev)
        for j in range(pool):
            mvk.server_eval(Ws[j], X[j], out=Y, stream=s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for k in range(reps):
            mvk.server_eval(Ws[k % pool], X[k % pool], out=Y, stream=s)

    def replay():
        with torch.cuda.stream(s):
            g.replay()

    warm(replay, args.warm_seconds)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(s):
        e0.record()
        g.replay()
        e1.record()
    torch.cuda.synchronize()
    t = 1e-3 * e0.elapsed_time(e1) / reps
    alg = m * n + 4 * n + 4 * m
    t_read = read_floor([w.data for w in Ws], reps, args)
    del Ws, X, Y, g
    torch.cuda.empty_cache()
    return {"workload": f"W {m}x{n} int8-valued, B=1, packed", "mean_launch_us": 1e6 * t,
            "achieved_gbps": alg / t / 1e9, "frac": alg / t / 1e9 / HBM_PEAK_GBS,
            "read_floor": {"mean_launch_us": 1e6 * t_read, "gbps": alg / t_read / 1e9, "frac": t_read / t}}


def server_eval_batched(args, gen, dev, m=28672, n=8192, B=64, pool=3, reps=30):
    """The batched kernel at 28672 x 8192 with 64 queries (235 MB of packed W per
    launch, a pool of three): HIP events around a graph of back-to-back
    launches; int8 matrix-core work 4 m n B multiply-adds (four digit planes)
    against the 5.0 POP/s dense int8 peak, and algorithmic HBM bytes."""
    import torch

    import paper_2609_10264_amd as mvk

    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        Ws = []
        for _ in range(pool):
            W = torch.randint(-127, 128, (m, n), generator=gen, device=dev, dtype=torch.int8)
            Ws.append(mvk.pack_weights(W, stream=s))
            del W
        X = torch.randint(0, mvk.P, (pool, B, n), generator=gen, device=dev, dtype=torch.int32)
        Y = torch.empty((B, m), dtype=torch.int32, device=dev)
        for j in range(pool):
            mvk.server_eval(Ws[j], X[j], out=Y, stream=s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for k in range(reps):
            mvk.server_eval(Ws[k % pool], X[k % pool], out=Y, stream=s)

    def replay():
        with torch.cuda.stream(s):
            g.replay()

    warm(replay, args.warm_seconds)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(s):
        e0.record()
        g.replay()
        e1.record()
    torch.cuda.synchronize()
    t = 1e-3 * e0.elapsed_time(e1) / reps
    alg = m * n + 4 * n * B + 4 * m * B
    ops = 2.0 * 4 * m * n * B
    del Ws, X, Y, g
    torch.cuda.empty_cache()
    return {"workload": f"W {m}x{n} int8-valued, B={B}, packed", "mean_launch_us": 1e6 * t,
            "modmac_per_s": m * n * B / t, "int8_tops": ops / t / 1e12,
            "mfma_frac": ops / t / MFMA_INT8_PEAK_OPS, "hbm_gbps": alg / t / 1e9}


def stack_bench(args):
    """32 decoder layers (seven projections each, 8 query columns): one step is a
    full pass (4 encodes, 7 server evaluations, 7 verifications per layer).
    Two schedules of the same work: serial (run_layer on one stream) and
    pipelined (prepare_layer for every layer on a preparation stream, flags
    ordering each layer's online part, run_layer_prepared, after its
    preparation); --mode picks the one reported as value."""
    import numpy as np
    import torch

    import paper_2609_10264_amd as mvk
    import paper_2609_10264_amd.stack as stack
    import synth

    cfg = synth.STACK
    layers, B, r, tx, ty, ell, cid = (cfg[k] for k in ("layers", "B", "r", "tx", "ty", "ell", "cid"))
    dev = torch.device("cuda")

    def d(a):
        return torch.from_numpy(np.ascontiguousarray(a).astype(np.int32)).to(dev)

    def make_code(kind, k):
        purpose = synth.PURPOSE_CX if kind == "x" else synth.PURPOSE_CY
        c = synth.raa_code(synth.seed_for(cid, purpose, sub=k), k, r)
        return mvk.Code(c["k"], c["r"], d(c["pi1"]), d(c["pi2"]), d(c["v1"]), d(c["v2"]))

    cx_by_n, cy_by_m = stack.codes_for(make_code)
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed)
    s = torch.cuda.Stream()
    built, inputs = [], []
    with torch.cuda.stream(s):
        for L in range(layers):
            Ws = {name: torch.randint(-127, 128, (m, n), generator=gen, device=dev, dtype=torch.int8)
                  for (name, m, n, _) in stack.PROJECTIONS}
            built.append(stack.build_layer(Ws, cx_by_n, cy_by_m))
            X = {grp: torch.randint(0, mvk.P, (B, stack.input_width(grp)), generator=gen, device=dev,
                                    dtype=torch.int32) for grp in stack.INPUTS}
            ex = {}
            for j, grp in enumerate(stack.INPUTS):
                i_, v_ = synth.sparse(synth.seed_for(cid, synth.PURPOSE_NOISE, 100 * L + j), B,
                                      r * stack.input_width(grp), tx)
                ex[grp] = (d(i_), d(v_))
            ey = {}
            for i, (name, m, _, _) in enumerate(stack.PROJECTIONS):
                i_, v_ = synth.sparse(synth.seed_for(cid, synth.PURPOSE_CHAL, 100 * L + i), ell, r * m, ty)
                ey[name] = (d(i_), d(v_))
            inputs.append((X, ex, ey))
    torch.cuda.synchronize()
    steps = max(1, args.steps // 40)
    warmup = max(1, args.warmup // 10)

    def time_graphs(replay, reps):
        warm(replay, args.warm_seconds)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            replay()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / reps

    # ---- serial -------------------------------------------------------------
    results = []

    def one_pass():
        results.clear()
        for L in range(layers):
            results.append(stack.run_layer(built[L], *inputs[L]))

    with torch.cuda.stream(s):
        for _ in range(warmup):
            one_pass()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        one_pass()

    def replay_serial():
        with torch.cuda.stream(s):
            g.replay()

    t_serial = time_graphs(replay_serial, steps)
    ok_serial = all(bool((out[name][1] == 1).all().item()) for out in results for name in out)
    last_serial = [t.clone() for t in results[-1]["down"][:2]]

    # ---- pipelined ----------------------------------------------------------
    s_prep, s_on = torch.cuda.Stream(), torch.cuda.Stream()
    nproj = len(stack.PROJECTIONS)
    flags = torch.zeros((layers, nproj), dtype=torch.int32, device=dev)
    late = torch.zeros((), dtype=torch.int32, device=dev)
    preps = [dict() for _ in range(layers)]
    presults = []

    def prep_pass():
        for L in range(layers):
            stack.prepare_layer(built[L], inputs[L][1], inputs[L][2], flags[L], out=preps[L], stream=s_prep)

    def online_pass():
        presults.clear()
        for L in range(layers):
            presults.append(stack.run_layer_prepared(built[L], inputs[L][0], preps[L], ready_flag=flags[L, nproj - 1],
                                                     timeout_us=200_000, timed_out=late, stream=s_on))

    for _ in range(warmup):  # also sizes the per-stream workspaces
        with torch.cuda.stream(s_prep):
            prep_pass()
        with torch.cuda.stream(s_on):
            online_pass()
        torch.cuda.synchronize()
    gp, go = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.graph(gp, stream=s_prep):
        prep_pass()
    with torch.cuda.graph(go, stream=s_on):
        online_pass()

    def replay_pipelined():
        # a pass's preparation starts after the previous pass's online part
        # (it rewrites the prepared buffers and the flags that part consumes),
        # and is submitted first: the two streams may share a hardware queue
        s_prep.wait_stream(s_on)
        with torch.cuda.stream(s_prep):
            gp.replay()
        with torch.cuda.stream(s_on):
            go.replay()

    late.zero_()
    t_pipe = time_graphs(replay_pipelined, steps)
    ok_pipe = all(bool((out[name][1] == 1).all().item()) for out in presults for name in out)
    ok_pipe = ok_pipe and int(late.item()) == 0
    same = all(bool(torch.equal(a, b)) for a, b in zip(last_serial, presults[-1]["down"][:2]))

    elapsed = t_pipe if args.mode == "pipelined" else t_serial
    macs = stack.macs_per_layer(B) * layers
    res = {"metric": METRIC, "value": macs / elapsed, "unit": "modMAC/s", "n_gpus": 1, "steps": steps,
           "warmup": warmup, "ms_per_step": 1e3 * elapsed, "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "i8xi8->i32 limb dot products, mod 2^31-1",
           "data": "synthetic",
           "config": {"workload": f"stack32: {layers} layers x (q,k,v,o 4096x4096; up,gate 11008x4096; "
                                  f"down 4096x11008), B={B}, r={r}, t_x={tx}, t_y={ty}, ell={ell}; step = one full "
                                  "pass (4 encodes, 7 server_evals, 7 decode_verifies per layer)",
                      "global_batch": B, "launch": "hip_graph", "mode": args.mode},
           "ms_per_step_pipelined": 1e3 * t_pipe, "ms_per_step_serial": 1e3 * t_serial,
           "all_accepted": ok_serial and ok_pipe, "pipelined_matches_one_call_path": same}
    print(json.dumps(res), flush=True)
    if not (ok_serial and ok_pipe and same):
        sys.exit(1)


def server_only(args, cfg, pool, total_steps, dev):
    """server_eval alone over a rotated pool of W, as a graph of back-to-back launches."""
    import numpy as np
    import torch

    import paper_2609_10264_amd as mvk

    m, n, B = cfg["m"], cfg["n"], cfg["B"]
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed)
    Ws = [torch.randint(-127, 128, (m, n), generator=gen, device=dev, dtype=torch.int8) for _ in range(pool)]
    if args.weights == "packed":
        Ws = [mvk.pack_weights(W) for W in Ws]
    X = torch.randint(0, mvk.P, (pool, B, n), generator=gen, device=dev, dtype=torch.int32)
    Y = torch.empty((B, m), dtype=torch.int32, device=dev)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        for i in range(max(args.warmup, pool)):
            mvk.server_eval(Ws[i % pool], X[i % pool], out=Y, path=args.path, stream=s)
    torch.cuda.synchronize()
    # K launches over the rotated pool captured as one HIP graph; HIP events on
    # the launch stream around its replay give the mean launch time.
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for i in range(args.steps):
            mvk.server_eval(Ws[i % pool], X[i % pool], out=Y, path=args.path, stream=s)
    def replay_g():
        with torch.cuda.stream(s):
            g.replay()

    warm(replay_g, args.warm_seconds)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    with torch.cuda.stream(s):
        e0.record()
        g.replay()
        e1.record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    mean_s = 1e-3 * e0.elapsed_time(e1) / args.steps
    ms = np.array([1e3 * mean_s])
    alg_bytes = m * n + 4 * n * B + 4 * m * B
    macs = m * n * B
    out = {"metric": METRIC, "value": macs / mean_s, "unit": "modMAC/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": 1e3 * elapsed / args.steps, "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "i8xi8->i32 limb dot products, mod 2^31-1",
           "data": "synthetic",
           "config": {"workload": f"{args.config}: server_eval only, W {m}x{n} int8-valued, B={B}",
                      "global_batch": B, "w_pool": pool, "weights": args.weights},
           "roofline": {"bound": "hbm", "achieved": alg_bytes / mean_s / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": alg_bytes / mean_s / 1e9 / HBM_PEAK_GBS, "traffic": None,
                        "kernel": f"server_eval ({args.path})", "alg_bytes_per_launch": alg_bytes,
                        "mean_launch_us": 1e6 * mean_s, "median_launch_us": 1e3 * float(np.median(ms))},
           "mfma_int8_tops": 2 * 4 * macs / mean_s / 1e12}
    print(json.dumps(out), flush=True)


def batch_verify_bench(args):
    """Batch verification of B claims M_b x_b = y_b (B matrices of the
    workload's shape, one verification code): the server's projection
    (mvk_batch_project) and the client's checks (mvk_batch_verify), against
    the client verifying the B claims one by one (mvk_verify, which gathers
    the rows of each Q_b itself).  Preprocessing untimed."""
    import numpy as np
    import torch

    import paper_2609_10264_amd as mvk
    import synth

    cfg = dict(synth.CONFIGS[args.config])
    m, n, r, ty, ell = (cfg[k] for k in ("m", "n", "r", "ty", "ell"))
    B, r2 = args.batch_verify, 2
    cid, dev = cfg["cid"], torch.device("cuda")

    def d(a):
        return torch.from_numpy(np.ascontiguousarray(a).astype(np.int32)).to(dev)

    def code(c):
        return mvk.Code(c["k"], c["r"], d(c["pi1"]), d(c["pi2"]), d(c["v1"]), d(c["v2"]))

    cx_h = synth.raa_code(synth.seed_for(cid, synth.PURPOSE_CX), n, r)
    cy_h = synth.raa_code(synth.seed_for(cid, synth.PURPOSE_CY), m, r)
    c2_h = synth.raa_code(synth.seed_for(cid, synth.PURPOSE_C2), B * n, r2)
    cx, cy, c2 = code(cx_h), code(cy_h), code(c2_h)
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed)
    Ws = [torch.randint(-127, 128, (m, n), generator=gen, device=dev, dtype=torch.int8) for _ in range(B)]
    keys = []
    for W in Ws:
        k = mvk.Key.allocate(m, n, cx, cy)
        mvk.keygen(k, W)
        keys.append(k)
    QtT, Qaux = mvk.batch_preprocess([k.Q for k in keys], c2)
    X = torch.randint(0, mvk.P, (B, n), generator=gen, device=dev, dtype=torch.int32)
    Y = torch.stack([mvk.server_eval(W, X[b:b + 1])[0] for b, W in enumerate(Ws)])
    steps = args.steps
    ei, ev = synth.sparse(synth.seed_for(cid, synth.PURPOSE_CHAL, 3), steps * ell, cy_h["N"], ty)
    e2i, e2v = synth.sparse(synth.seed_for(cid, synth.PURPOSE_CHAL2, 3), steps * ell, c2_h["N"], ty)
    EI, EV = d(ei).view(steps, ell, ty), d(ev).view(steps, ell, ty)
    E2I, E2V = d(e2i).view(steps, ell, ty), d(e2v).view(steps, ell, ty)
    Ut = torch.empty((steps, ell, B * n), dtype=torch.int32, device=dev)
    acc = torch.zeros((steps, B), dtype=torch.int32, device=dev)
    acc1 = torch.zeros((steps, B), dtype=torch.int32, device=dev)
    s = torch.cuda.Stream()

    def one_batch(i):
        mvk.batch_project(QtT, n, EI[i], EV[i], out=Ut[i])
        mvk.batch_verify(cy, c2, Qaux, X, Y, EI[i], EV[i], Ut[i], E2I[i], E2V[i], accept=acc[i])

    def one_by_one(i):
        for b in range(B):
            mvk.verify(keys[b], X[b:b + 1], Y[b:b + 1], EI[i], EV[i], accept=acc1[i, b:b + 1])

    out = {}
    for name, fn in (("batch", one_batch), ("one_by_one", one_by_one)):
        with torch.cuda.stream(s):
            fn(0)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for i in range(steps):
                fn(i)

        def replay():
            with torch.cuda.stream(s):
                g.replay()

        warm(replay, args.warm_seconds)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(s):
            e0.record()
            g.replay()
            e1.record()
        torch.cuda.synchronize()
        out[name] = 1e3 * e0.elapsed_time(e1) / steps
    ok = bool((acc == 1).all().item()) and bool((acc1 == 1).all().item())
    res = {"metric": "batch verification time per batch of claims (Protocol Batch-vMVMD), 1×MI355X",
           "value": out["batch"], "unit": "us", "n_gpus": 1, "steps": steps, "warmup": args.warmup,
           "higher_is_better": False, "data": "synthetic",
           "config": {"workload": f"{B} claims of W {m}x{n} (int8-valued in F_p), primary RAA r={r}, "
                                  f"secondary RAA r'={r2} over Bn={B * n}, t=t'={ty}, ell=ell'={ell}",
                      "claims": B},
           "batch_us": out["batch"], "one_by_one_us": out["one_by_one"], "all_accepted": ok}
    print(json.dumps(res), flush=True)
    if not ok:
        sys.exit(1)


# The paper's own timings for this workload (Sec. 7.1, online-breakdown and
# preprocessing tables; Rust, one thread of an x86 c8i.4xlarge, BabyBear):
# n -> (server MVM, client online total, one-time preprocessing), milliseconds.
PAPER_SEC71_MS = {1024: (0.39, 0.79, 329.54), 2048: (1.59, 1.55, 1499.06), 4096: (9.54, 2.33, 6030.76),
                  8192: (34.68, 4.56, 25063.59), 16384: (116.00, 9.33, 135800.06)}


def paper_eval_bench(args):
    """The pvMVMD evaluation of Sec. 7.1 on the GPU, over BabyBear: square
    n x n int8-valued W, one query, RAA rate 1/8 for both codes, t_x of Eq. (1),
    t_y = 31, ell = 2, for n = 2^10 .. 2^14 (or --n).  Per n: keygen (P^T and Q,
    the one-time preprocessing), and HIP-event means over graphs of K calls of
    encode, server_eval and decode_verify alone and of the whole step, cycling a
    pool of distinct W (and keys) that exceeds the last-level cache twice."""
    import numpy as np
    import torch

    import oracle
    import paper_2609_10264_amd as mvk
    import synth

    cfg = synth.PAPER_EVAL
    p, r, ty, ell, B, cid = (cfg[k] for k in ("p", "r", "ty", "ell", "B", "cid"))
    dev = torch.device("cuda")
    s = torch.cuda.Stream()
    K = max(8, args.steps)
    ns = [args.n] if args.n else sorted(cfg["tx"])

    def d(a):
        return torch.from_numpy(np.ascontiguousarray(a).astype(np.int32)).to(dev)

    def code(c):
        return mvk.Code(c["k"], c["r"], d(c["pi1"]), d(c["pi2"]), d(c["v1"]), d(c["v2"]), p)

    def timed(fn, reps):
        """Mean milliseconds per call of fn(i), i < reps, from one graph replay."""
        with torch.cuda.stream(s):
            fn(0)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for i in range(reps):
                fn(i)

        def replay():
            with torch.cuda.stream(s):
                g.replay()

        warm(replay, args.warm_seconds)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(s):
            e0.record()
            g.replay()
            e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    rows, ok = [], True
    for n in ns:
        m, tx = n, cfg["tx"][n]
        pool = max(2, -(-2 * 256 * 2**20 // (m * n)))
        cx_h = synth.raa_code(synth.seed_for(cid, synth.PURPOSE_CX, n), n, r, p=p)
        cy_h = synth.raa_code(synth.seed_for(cid, synth.PURPOSE_CY, n), m, r, p=p)
        cx, cy = code(cx_h), code(cy_h)
        gen = torch.Generator(device=dev)
        gen.manual_seed(args.seed + n)
        Ws, keys, kg_ms = [], [], []
        with torch.cuda.stream(s):
            for j in range(pool + 1):  # the first keygen (workspace sizing) is not timed
                Wj = torch.randint(-127, 128, (m, n), generator=gen, device=dev, dtype=torch.int8)
                kj = mvk.Key.allocate(m, n, cx, cy)
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                mvk.keygen(kj, Wj, stream=s)
                e1.record()
                e1.synchronize()
                if j:
                    kg_ms.append(e0.elapsed_time(e1))
                    Ws.append(mvk.pack_weights(Wj, stream=s))
                    keys.append(kj)
                del Wj
        X = torch.randint(0, p, (K, B, n), generator=gen, device=dev, dtype=torch.int32)
        exi, exv = synth.sparse(synth.seed_for(cid, synth.PURPOSE_NOISE, n), K * B, cx.N, tx, p=p)
        eyi, eyv = synth.sparse(synth.seed_for(cid, synth.PURPOSE_CHAL, n), K * ell, cy.N, ty, p=p)
        EXI, EXV = d(exi).view(K, B, tx), d(exv).view(K, B, tx)
        EYI, EYV = d(eyi).view(K, ell, ty), d(eyv).view(K, ell, ty)
        Xh = torch.empty((K, B, n), dtype=torch.int32, device=dev)
        Yh = torch.empty((K, B, m), dtype=torch.int32, device=dev)
        Y = torch.empty((K, B, m), dtype=torch.int32, device=dev)
        ACC = torch.zeros((K, B), dtype=torch.int32, device=dev)

        def enc(i):
            mvk.encode(keys[i % pool], X[i], EXI[i], EXV[i], out=Xh[i])

        def se(i):
            mvk.server_eval(Ws[i % pool], Xh[i], out=Yh[i], p=p)

        def dv(i):
            mvk.decode_verify(keys[i % pool], Xh[i], Yh[i], EXI[i], EXV[i], EYI[i], EYV[i], Y=Y[i], accept=ACC[i])

        def step(i):
            enc(i)
            se(i)
            dv(i)

        t_enc, t_se, t_dv = timed(enc, K), timed(se, K), timed(dv, K)
        ACC.zero_()
        t_step = timed(step, K)
        acc_ok = bool((ACC == 1).all().item())
        # boost mode (Sec. 7): the masks and challenge vectors of every step
        # prepared ahead (client_prepare, timed on its own); online only
        # encode_masked -> server_eval -> decode_verify_masked
        preps = [mvk.Prepared(keys[i % pool], B, ell) for i in range(K)]

        def prep(i):
            mvk.client_prepare(keys[i % pool], EXI[i], EXV[i], EYI[i], EYV[i], out=preps[i])

        def online(i):
            mvk.encode_masked(keys[i % pool], X[i], preps[i], out=Xh[i])
            se(i)
            mvk.decode_verify_masked(keys[i % pool], Xh[i], Yh[i], preps[i], Y=Y[i], accept=ACC[i])

        t_prep = timed(prep, K)
        ACC.zero_()
        t_online = timed(online, K)
        acc_ok = acc_ok and bool((ACC == 1).all().item())
        del preps
        # the last step's decrypted output against the server product of the plaintext query
        with torch.cuda.stream(s):
            plain = mvk.server_eval(Ws[(K - 1) % pool], X[K - 1], p=p)
        torch.cuda.synchronize()
        acc_ok = acc_ok and bool(torch.equal(plain, Y[K - 1]))
        ok = ok and acc_ok
        alg_bytes = m * n + 4 * n * B + 4 * m * B
        srv_s = 1e-3 * t_se
        paper = PAPER_SEC71_MS[n]
        rows.append({"n": n, "t_x": tx, "w_pool": pool, "keygen_ms": float(np.mean(kg_ms)),
                     "encode_us": 1e3 * t_enc, "server_eval_us": 1e3 * t_se, "decode_verify_us": 1e3 * t_dv,
                     "step_us": 1e3 * t_step, "boost_prepare_us": 1e3 * t_prep, "boost_online_us": 1e3 * t_online,
                     "server_gb_per_s": alg_bytes / srv_s / 1e9,
                     "server_hbm_frac": alg_bytes / srv_s / 1e9 / HBM_PEAK_GBS,
                     "step_modmac_per_s": m * n * B / (1e-3 * t_step), "all_accepted": acc_ok,
                     "paper_cpu_ms": {"server": paper[0], "client_online": paper[1], "preprocessing": paper[2]}})
        del Ws, keys, X, Xh, Yh, Y
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    top = rows[-1]
    res = {"metric": METRIC, "value": top["step_modmac_per_s"], "unit": "modMAC/s", "n_gpus": 1, "steps": K,
           "warmup": 1, "ms_per_step": 1e-3 * top["step_us"], "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "i8xi8->i32 limb dot products, mod 15*2^27+1", "data": "synthetic",
           "config": {"workload": f"Sec. 7.1 pvMVMD evaluation over BabyBear: W {top['n']}x{top['n']} int8-valued, "
                                  f"one query, RAA r={r}, t_x={top['t_x']}, t_y={ty}, ell={ell}; step = "
                                  "encode+server_eval+decode_verify", "global_batch": B, "launch": "hip_graph"},
           "sweep": rows, "all_accepted": ok}
    if not args.no_cpu_baseline:
        # the oracle's server product over a row sample of the largest W
        n = top["n"]
        Wh = synth.weights(synth.seed_for(cid, synth.PURPOSE_W, n), 256, n)
        Xq = synth.field_uniform(synth.seed_for(cid, synth.PURPOSE_X, n), (1, n), p=p)
        reps, el = 0, 0.0
        while el < min(args.cpu_seconds, 5.0):
            t0 = time.perf_counter()
            oracle.server_eval(Wh, Xq, p=p)
            el += time.perf_counter() - t0
            reps += 1
        res["cpu_baseline"] = {"value": 256 * n * reps / el, "unit": "modMAC/s", "cores": 1, "kind": "oracle",
                               "host_cpu": host_cpu(),
                               "sample": f"{reps} oracle server products of 256 rows x {n} over BabyBear, "
                                         f"{el:.1f} s; single-threaded C, '%' per field op"}
    print(json.dumps(res), flush=True)
    if not ok:
        sys.exit(1)


def host_cpu() -> str:
    """The host CPU model (Linux /proc/cpuinfo), for the CPU baseline's record."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


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
    return {"value": m * n * B * steps / el, "unit": "modMAC/s", "cores": 1, "kind": "oracle", "host_cpu": host_cpu(),
            "sample": f"{steps} full steps (encode+server_eval+verify+decode) of the same workload, one W, "
                      f"{el:.1f} s of oracle time (input drawing excluded); single-threaded C, '%' per field op"}


if __name__ == "__main__":
    main()
