"""Benchmark of the pvMVMD hot path on one MI355X.

Default run (the line the driver reads): the 32-layer decoder stack, the
largest workload that fits one GPU.  Per layer seven projections (q, k, v, o
4096 x 4096; up, gate 11008 x 4096; down 4096 x 11008, int8-valued W over
p = 2^31 - 1), eight query columns, RAA r = 3, t_x = 64, t_y = 31, ell = 2.
One step = one pass over the 32 layers: per layer 4 encodes (Encrypt:
x^ = x + Gx e_x), 7 server products (y^ = W x^ mod p) and 7 decode/verify
calls (Verify with ell sparse challenges + Decrypt), with one response in
1000 tampered (a nonzero delta at a seeded coordinate) and rejected inside
the timed region.  Every input (6.48 GB of packed W, 155 GB of P^T and Q, the
queries, noise and challenges) is resident in HBM before timing.

Three schedules of the same work (--stack-mode):
  overlapped  the paper's standard mode with precomputation
              (Sec. 7): the work that depends on neither the query nor the
              response (masks Gx e_x and P e_x, challenge vectors Gy e_q and
              e_q^T Q; client_prepare) runs on preparation streams one layer
              ahead; the online part (encode_masked -> server_eval ->
              decode_verify_masked) keeps the order of an inference pass (q, k,
              v, then o, then up and gate, then down, each input after the
              previous stage's checks) with the projections of a stage side by
              side.  One HIP graph of the pass over several streams.
  pipelined   (default) the same work on preparation streams (one graph
              each, every input's preparation one launch for the projections
              it feeds) and one online stream (per input in inference order:
              masked encode, one grouped server launch, one grouped check),
              with a device flag per input between the graphs.
  serial      every call of the pass back to back on one stream, one graph.

The JSON line:
  value       modMAC/s of the whole pass (51.8 G mod-MACs / pass time), in the
              chosen schedule; every schedule's pass time beside it
  roofline    the pass's 128 server calls (per layer: q, k, v grouped in one
              launch over their shared input, o, up and gate grouped, down),
              captured back to back as a graph and timed with HIP events on
              their stream: algorithmic bytes (m*n + 4*n*B + 4*m*B per
              product) over their device time, against 8 TB/s of HBM; per
              call type beside it, and a streaming read of the same W buffers
              (the measured read floor)
  cpu_baseline the CPU oracle (plain C, threaded over row blocks on every core
              of this host) on one layer's step of the same shapes
  configs     the single-matrix workloads (4096 x 4096 B=1, 11008 x 4096 B=16,
              28672 x 8192 B=64), each with its own step time, roofline and
              cpu_baseline
--config <name> runs one workload alone; --config paper_eval the Sec. 7.1
sweep over BabyBear; --batch-verify B batch verification.
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
KERNEL_SRC = os.path.join(ROOT, "paper_2609_10264_amd", "csrc", "server_eval.hip")
STACK_LAUNCHES_PER_PASS = 32 * 4  # server calls per pass: (q,k,v), o, (up,gate), down per layer
SIDE_CONFIGS = ("attn4096", "mlp_up_11008x4096", "mlp_large_28672x8192")
DTYPE = "i8xi8->i32 limb dot products, mod 2^31-1"


def kernel_src_sha256() -> str:
    import hashlib
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def traffic_file(config: str) -> str:
    return os.path.join(ROOT, "profiles", f"server_eval_{config}_traffic.json")


def measured_traffic(config: str, weights: str):
    """HBM bytes per server_eval launch (per pass of the 128 server calls for the
    stack) from the committed counter runs, if they were taken on the current
    kernel source, this workload and weight layout; else None."""
    try:
        with open(traffic_file(config)) as f:
            rec = json.load(f)
        sha = kernel_src_sha256()
    except OSError:
        return None
    if rec.get("kernel_src_sha256") != sha or rec.get("config") != config or rec.get("weights") != weights:
        return None
    return rec.get("traffic_bytes_per_launch")


def write_traffic(fetch_csv: str, write_csv: str, config: str, weights: str, copy_mib: int, kernel_match: str):
    """Traffic record from two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE; KiB
    per dispatch) of `bench.py --calib-copy-mib copy_mib`, each scaled by what
    the same counter reads for the copy_mib MiB device copy (which reads and
    writes copy_mib MiB).  Single-matrix workloads: the median over the
    dispatches whose name contains kernel_match.  The stack: the sum over
    those dispatches divided by the passes they make up (128 per pass)."""
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
        if config == "stack32":
            passes = len(vals) / STACK_LAUNCHES_PER_PASS
            return sum(vals) / passes, len(vals), max(copies)
        return statistics.median(vals), len(vals), max(copies)

    f_med, f_n, f_copy = per_kernel(fetch_csv, "FETCH_SIZE")
    w_med, w_n, w_copy = per_kernel(write_csv, "WRITE_SIZE")
    ref_kib = copy_mib * 1024.0
    fs, ws = ref_kib / f_copy, ref_kib / w_copy
    unit = "pass" if config == "stack32" else "dispatch"
    rec = {"kernel": kernel_match, "config": config, "weights": weights, "kernel_src_sha256": kernel_src_sha256(),
           f"fetch_size_kib_per_{unit}": f_med, f"write_size_kib_per_{unit}": w_med, "dispatches": [f_n, w_n],
           "copy_reference_mib": copy_mib, "copy_fetch_size_kib": f_copy, "copy_write_size_kib": w_copy,
           "fetch_scale": fs, "write_scale": ws,
           "traffic_bytes_per_launch": int(round((f_med * fs + w_med * ws) * 1024))}
    with open(traffic_file(config), "w") as f:
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


def graph_mean_seconds(stream, body, reps, warm_seconds, prime=None):
    """Mean seconds per call of body(k), k < reps, captured back to back as one
    HIP graph on `stream` and timed with HIP events on that stream."""
    import torch

    with torch.cuda.stream(stream):
        (prime or body)(0)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for k in range(reps):
            body(k)

    def replay():
        with torch.cuda.stream(stream):
            g.replay()

    warm(replay, warm_seconds)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        e0.record()
        g.replay()
        e1.record()
    torch.cuda.synchronize()
    del g
    return 1e-3 * e0.elapsed_time(e1) / reps


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20, help="timed steps of the headline workload")
    ap.add_argument("--warmup", type=int, default=5, help="untimed steps before them")
    ap.add_argument("--config", default="all",
                    help="all (the stack line with the single-matrix workloads as side keys), stack32, one of "
                         "synth.CONFIGS, or paper_eval")
    ap.add_argument("--side-steps", type=int, default=100, help="timed steps of each single-matrix side workload")
    ap.add_argument("--side-warmup", type=int, default=10)
    ap.add_argument("--pool", type=int, default=0, help="distinct W matrices cycled (0: enough for 2x the LLC)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="oracle time of the headline CPU baseline")
    ap.add_argument("--side-cpu-seconds", type=float, default=4.0, help="oracle time of each side CPU baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-side", action="store_true", help="headline only")
    ap.add_argument("--no-large", action="store_true", help="skip the 16384 x 16384 single-query measurement")
    ap.add_argument("--eager", action="store_true", help="launch the timed steps one by one instead of a HIP graph")
    ap.add_argument("--chains", type=int, default=1,
                    help="serial mode of a single-matrix workload: independent query chains on their own streams")
    ap.add_argument("--mode", default="pipelined", choices=["pipelined", "serial"],
                    help="schedule reported as value of a single-matrix workload (both are timed)")
    ap.add_argument("--stack-mode", default="pipelined", choices=["overlapped", "pipelined", "serial"],
                    help="schedule reported as value of the stack (all three are timed)")
    ap.add_argument("--prep-streams", type=int, default=1,
                    help="preparation streams of the pipelined and overlapped stack schedules (more than one "
                         "measured slower: 5.4 against 4.2 ms per pass with two)")
    ap.add_argument("--prep-cus", type=int, default=64,
                    help="pipelined stack schedule: compute units of the preparation stream (the online stream "
                         "gets the others; 0: both streams on every unit). Measured 3.69 ms per pass with 64, "
                         "4.00 ms with 0")
    ap.add_argument("--config-prep-cus", type=int, default=0,
                    help="the same split for the single-matrix workloads' pipelined schedule (0: none; with 64 "
                         "their preparation, which outweighs the server call at 11008x4096 B=16 and "
                         "28672x8192 B=64, became the bound)")
    ap.add_argument("--client-turn", type=int, default=1, choices=[0, 1],
                    help="single-matrix pipelined schedule: one launch per step for the response's "
                         "decode/verify and the next query's masked encode (1), or separate launches (0)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after the run, copy a buffer of this many MiB (reference for the traffic counters)")
    ap.add_argument("--seed", type=int, default=2609)
    ap.add_argument("--warm-seconds", type=float, default=0.3,
                    help="untimed graph replays before each timed replay (clock ramp-up)")
    ap.add_argument("--path", default="auto", choices=["auto", "valu", "mfma"], help="server_eval kernel family")
    ap.add_argument("--write-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="derive the traffic record of --config from two rocprofv3 --pmc counter files and exit")
    ap.add_argument("--traffic-kernel", default="server_eval_mfma",
                    help="kernel-name substring selected by --write-traffic")
    ap.add_argument("--weights", default="packed", choices=["packed", "rowmajor"],
                    help="server-side layout of W (packed: matrix-core operand order, written once like P^T and Q)")
    ap.add_argument("--m", type=int, default=0, help="override the workload's row count (server-only)")
    ap.add_argument("--n", type=int, default=0, help="override the workload's column count (server-only)")
    ap.add_argument("--B", type=int, default=0, help="override the workload's query count (server-only)")
    ap.add_argument("--server-only", action="store_true",
                    help="time server_eval alone over a rotated W pool (no client steps)")
    ap.add_argument("--batch-verify", type=int, default=0, metavar="B",
                    help="time batch verification (Protocol Batch-vMVMD) of B claims of the workload's shape")
    return ap.parse_args()


def main():
    args = parse()
    if args.write_traffic:
        cfg = "stack32" if args.config in ("all", "stack32") else args.config
        return write_traffic(args.write_traffic[0], args.write_traffic[1], cfg, args.weights,
                             args.calib_copy_mib or 256, args.traffic_kernel)
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; runs on several GPUs are not supported",
                          "n_gpus": args.gpus}), flush=True)
        sys.exit(2)

    import torch

    import synth

    torch.cuda.set_device(0)
    if args.batch_verify:
        return batch_verify_bench(args)
    if args.config == "paper_eval":
        return paper_eval_bench(args)
    if args.server_only:
        cfg = dict(synth.CONFIGS[args.config])
        for key in ("m", "n", "B"):
            if getattr(args, key):
                cfg[key] = getattr(args, key)
        pool = args.pool or max(2, -(-2 * 256 * 2**20 // (cfg["m"] * cfg["n"])))
        return server_only(args, cfg, pool, args.warmup + args.steps, torch.device("cuda"))
    if args.config in synth.CONFIGS:
        res = config_bench(args, args.config, args.steps, args.warmup, args.cpu_seconds, large=not args.no_large)
        ok = res.pop("_ok")
    else:
        if args.config not in ("all", "stack32"):
            raise SystemExit(f"unknown --config {args.config}")
        res = stack_bench(args, args.steps, args.warmup, args.cpu_seconds)
        ok = res.pop("_ok")
        if args.config == "all" and not args.no_side:
            torch.cuda.synchronize()
            torch.cuda.empty_cache()
            side = {}
            for name in SIDE_CONFIGS:
                print(f"[bench] side workload {name}", file=sys.stderr, flush=True)
                side[name] = config_bench(args, name, args.side_steps, args.side_warmup, args.side_cpu_seconds,
                                          large=(name == "attn4096" and not args.no_large))
                ok = side[name].pop("_ok") and ok
                torch.cuda.synchronize()
                torch.cuda.empty_cache()
            res["configs"] = side
    if args.calib_copy_mib:
        calib_copy(args.calib_copy_mib)
    print(json.dumps(res), flush=True)
    if not ok:
        sys.exit(1)


def config_bench(args, name, steps, warmup, cpu_seconds, large=False):
    """One single-matrix workload: K whole steps (encode -> server_eval ->
    decode_verify) in both schedules over a pool of distinct W (each with its
    own P^T and Q) that exceeds the last-level cache twice, the server_eval
    roofline, and the oracle's CPU baseline.  Returns the record (with "_ok")."""
    import numpy as np
    import torch

    import paper_2609_10264_amd as mvk
    import synth

    cfg = dict(synth.CONFIGS[name])
    m, n, B, r, tx, ty, ell = (cfg[k] for k in ("m", "n", "B", "r", "tx", "ty", "ell"))
    cid = cfg["cid"]
    pool = args.pool or max(2, -(-2 * 256 * 2**20 // (m * n)))
    total_steps = warmup + steps
    dev = torch.device("cuda")

    def d(a):
        a = np.ascontiguousarray(a)
        return torch.from_numpy(a.astype(np.int32) if a.dtype != np.int8 else a).to(dev)

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
        del Wj
    X = torch.randint(0, mvk.P, (total_steps, B, n), generator=gen, device=dev, dtype=torch.int32)
    exi, exv = synth.sparse(synth.seed_for(cid, synth.PURPOSE_NOISE, 7), total_steps * B, cx.N, tx)
    eyi, eyv = synth.sparse(synth.seed_for(cid, synth.PURPOSE_CHAL, 7), total_steps * ell, cy.N, ty)
    EXI, EXV = d(exi).view(total_steps, B, tx), d(exv).view(total_steps, B, tx)
    EYI, EYV = d(eyi).view(total_steps, ell, ty), d(eyv).view(total_steps, ell, ty)
    C = max(1, args.chains)
    if warmup < C:
        raise SystemExit("--warmup must be at least --chains (each chain warms its own stream)")
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
    for i in range(warmup):
        with torch.cuda.stream(streams[i % C]):
            step(i)
    torch.cuda.synchronize()
    timed = [[warmup + k for k in range(steps) if (warmup + k) % C == c] for c in range(C)]

    if args.eager:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(steps):
            i = warmup + k
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
    accepted = bool((ACC[warmup:] == 1).all().item())
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
    cu_streams = []
    if args.config_prep_cus:  # preparation and online calls on disjoint compute units
        ncu = mvk.device_cus()
        if not 0 < args.config_prep_cus < ncu:
            raise SystemExit(f"--config-prep-cus must be between 1 and {ncu - 1}")
        cu_streams = [mvk.CUStream(0, args.config_prep_cus),
                      mvk.CUStream(args.config_prep_cus, ncu - args.config_prep_cus)]
        s_prep, s_on = cu_streams[0].stream, cu_streams[1].stream
    else:
        s_prep, s_on = torch.cuda.Stream(), torch.cuda.Stream()
    pXhs = [torch.empty((B, n), dtype=torch.int32, device=dev) for _ in range(2)]
    pXh = pXhs[0]
    pYh = torch.empty((B, m), dtype=torch.int32, device=dev)
    pY = torch.empty((B, m), dtype=torch.int32, device=dev)

    def prepare(i):
        j = i % pool
        mvk.client_prepare(keys[j], EXI[i], EXV[i], EYI[i], EYV[i], out=preps[i], done_flag=flags[i])

    def online(seq):
        """The online part of the steps in seq.  Client turns (default): the
        first masked encode, then per step the server call and one launch
        with this response's decode/verify and the next query's masked encode
        (the queries are independent), two X^ buffers in turn; else three
        launches per step."""
        if not args.client_turn or not seq:
            for i in seq:
                j = i % pool
                mvk.encode_masked(keys[j], X[i], preps[i], out=pXh, ready_flag=flags[i], timeout_us=50_000,
                                  timed_out=late)
                mvk.server_eval(Ws[j], pXh, out=pYh, path=args.path)
                mvk.decode_verify_masked(keys[j], pXh, pYh, preps[i], Y=pY, accept=ACC2[i])
            return pXh
        i0 = seq[0]
        mvk.encode_masked(keys[i0 % pool], X[i0], preps[i0], out=pXhs[0], ready_flag=flags[i0], timeout_us=50_000,
                          timed_out=late)
        for k, i in enumerate(seq):
            j, cur = i % pool, pXhs[k % 2]
            mvk.server_eval(Ws[j], cur, out=pYh, path=args.path)
            if k + 1 < len(seq):
                i1 = seq[k + 1]
                mvk.decode_verify_encode_masked(keys[j], cur, pYh, preps[i], X[i1], preps[i1], Y=pY, accept=ACC2[i],
                                                out_next=pXhs[(k + 1) % 2], ready_flag=flags[i1], timeout_us=50_000,
                                                timed_out=late)
            else:
                mvk.decode_verify_masked(keys[j], cur, pYh, preps[i], Y=pY, accept=ACC2[i])
        return pXhs[(len(seq) - 1) % 2]

    for i in range(warmup):  # also sizes the library's per-stream workspaces
        with torch.cuda.stream(s_prep):
            prepare(i)
    with torch.cuda.stream(s_on):
        online(list(range(warmup)))
    torch.cuda.synchronize()
    steps_t = list(range(warmup, total_steps))
    g_prep, g_on = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_prep, stream=s_prep):
        for i in steps_t:
            prepare(i)
    with torch.cuda.graph(g_on, stream=s_on):
        last_xh = online(steps_t)

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
    accepted_pipe = bool((ACC2[warmup:] == 1).all().item()) and int(late.item()) == 0
    # the last timed step again through the one-call path: same Xhat, Yhat, Y
    i_last = steps_t[-1]
    got = (last_xh.clone(), pYh.clone(), pY.clone())
    with torch.cuda.stream(s_on):
        rXh = mvk.encode(keys[i_last % pool], X[i_last], EXI[i_last], EXV[i_last])
        rYh = mvk.server_eval(Ws[i_last % pool], rXh, path=args.path)
        rY, _, _, _ = mvk.decode_verify(keys[i_last % pool], rXh, rYh, EXI[i_last], EXV[i_last], EYI[i_last],
                                        EYV[i_last])
    torch.cuda.synchronize()
    pipe_matches = all(bool(torch.equal(a, b)) for a, b in zip(got, (rXh, rYh, rY)))
    del g_prep, g_on, preps
    for c in cu_streams:
        c.close()
    if not args.eager:
        del graphs
    elapsed = elapsed_pipe if args.mode == "pipelined" else elapsed_serial

    # server_eval alone over the same W pool, captured back to back; HIP events
    # on the launch stream bracket the replay.
    s = streams[0]
    reps = max(steps, 2 * pool)
    Xs = torch.randint(0, mvk.P, (pool, B, n), generator=gen, device=dev, dtype=torch.int32)
    se_mean_s = graph_mean_seconds(s, lambda k: mvk.server_eval(Ws[k % pool], Xs[k % pool], out=Yh[0],
                                                                 path=args.path), reps, args.warm_seconds)
    read_s = read_floor([w.data if isinstance(w, mvk.PackedW) else w for w in Ws], reps, args)
    macs = m * n * B
    alg_bytes = m * n + 4 * n * B + 4 * m * B
    achieved = alg_bytes / se_mean_s / 1e9
    out = {
        "workload": f"{name}: W {m}x{n} int8-valued in F_p (p=2^31-1), B={B} query column(s), RAA r={r}, "
                    f"t_x={tx}, t_y={ty}, ell={ell}; step = encode+server_eval+decode_verify",
        "value": macs * steps / elapsed, "unit": "modMAC/s", "steps": steps, "warmup": warmup,
        "ms_per_step": 1e3 * elapsed / steps, "mode": args.mode,
        "ms_per_step_pipelined": 1e3 * elapsed_pipe / steps, "ms_per_step_serial": 1e3 * elapsed_serial / steps,
        "prep_cus": args.config_prep_cus, "client_turn": bool(args.client_turn),
        "w_pool": pool, "weights": args.weights, "launch": "eager" if args.eager else "hip_graph",
        "chains": C if args.mode == "serial" else 1,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": measured_traffic(name, args.weights),
                     "kernel": f"server_eval ({args.path})", "alg_bytes_per_launch": alg_bytes,
                     "mean_launch_us": 1e6 * se_mean_s, "launches": reps,
                     "read_floor": {"mean_launch_us": 1e6 * read_s, "gbps": alg_bytes / read_s / 1e9,
                                    "frac": read_s / se_mean_s}},
        "server_eval": {"modmac_per_s": macs / se_mean_s, "gb_per_s": achieved},
        "all_accepted": accepted_serial and accepted_pipe,
        "replay_matches_eager": replay_matches_eager,
        "pipelined_matches_one_call_path": pipe_matches,
    }
    if B > 4:
        ops = 2.0 * 4 * macs  # four int8 digit planes per mod-MAC
        out["mfma"] = {"int8_tops": ops / se_mean_s / 1e12, "peak_tops": MFMA_INT8_PEAK_OPS / 1e12,
                       "frac": ops / se_mean_s / MFMA_INT8_PEAK_OPS,
                       "ops_per_alg_byte": ops / alg_bytes, "ridge_ops_per_byte": MFMA_INT8_PEAK_OPS / 8e12}
    del Ws, keys, X, Xs
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    if large:
        out["server_eval_large"] = server_eval_large(args, gen, dev)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_config(cfg, cpu_seconds)
    out["_ok"] = accepted_serial and accepted_pipe and replay_matches_eager and pipe_matches
    return out


def stack_bench(args, steps, warmup, cpu_seconds):
    """The 32-layer stack (seven projections per layer, 8 query columns): one
    step is a full pass (4 encodes, 7 server evaluations, 7 verifications per
    layer) with the seeded one-in-1000 tampered responses.  Both schedules are
    timed over `steps` passes after `warmup` untimed ones; returns the record
    (with "_ok")."""
    import numpy as np
    import torch

    import paper_2609_10264_amd as mvk
    import paper_2609_10264_amd.stack as stack
    import synth

    cfg = synth.STACK
    layers, B, r, tx, ty, ell, cid = (cfg[k] for k in ("layers", "B", "r", "tx", "ty", "ell", "cid"))
    nproj = len(stack.PROJECTIONS)
    dev = torch.device("cuda")
    P = mvk.P

    def d(a):
        return torch.from_numpy(np.ascontiguousarray(a).astype(np.int32)).to(dev)

    def make_code(kind, k):
        purpose = synth.PURPOSE_CX if kind == "x" else synth.PURPOSE_CY
        c = synth.raa_code(synth.seed_for(cid, purpose, sub=k), k, r)
        return mvk.Code(c["k"], c["r"], d(c["pi1"]), d(c["pi2"]), d(c["v1"]), d(c["v2"]))

    t_setup = time.perf_counter()
    cx_by_n, cy_by_m = stack.codes_for(make_code)
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed)
    s = torch.cuda.Stream()
    built, inputs, pre_ms = [], [], []
    with torch.cuda.stream(s):
        for L in range(layers):
            Ws = {name: torch.randint(-127, 128, (m, n), generator=gen, device=dev, dtype=torch.int8)
                  for (name, m, n, _) in stack.PROJECTIONS}
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            built.append(stack.build_layer(Ws, cx_by_n, cy_by_m, stream=s))
            e1.record(s)
            e1.synchronize()
            if L:  # the first layer sizes the workspace
                pre_ms.append(e0.elapsed_time(e1))
            del Ws
            X = {grp: torch.randint(0, P, (B, stack.input_width(grp)), generator=gen, device=dev,
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
    t_setup = time.perf_counter() - t_setup
    print(f"[bench] stack setup {t_setup:.1f} s", file=sys.stderr, flush=True)

    # one response in 1000 of a pass (layer, projection, column) is tampered
    total = layers * nproj * B
    g = synth.rng(synth.seed_for(cid, synth.PURPOSE_TAMPER))
    offset = int(g.integers(0, 1000))
    plan = {}
    for k in range(offset, total, 1000):
        L, rest = divmod(k, nproj * B)
        i, b = divmod(rest, B)
        m = stack.PROJECTIONS[i][1]
        plan.setdefault((L, stack.PROJECTIONS[i][0]), []).append((b, int(g.integers(0, m)), int(g.integers(1, P))))

    def tamperer(L):
        def tamper(name, Yhat):
            for b, pos, delta in plan.get((L, name), []):
                Yhat[b, pos] = (Yhat[b, pos].to(torch.int64) + delta) % P
        return tamper

    def expected_accept(L, name):
        bad = {b for (b, _, _) in plan.get((L, name), [])}
        return [0 if b in bad else 1 for b in range(B)]

    def accepts_ok(results):
        return all(out[name][1].tolist() == expected_accept(L, name)
                   for L, out in enumerate(results) for name in out)

    def time_passes(replay):
        warm(replay, args.warm_seconds)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            replay()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / steps

    # ---- serial -------------------------------------------------------------
    results = []

    def one_pass():
        results.clear()
        for L in range(layers):
            results.append(stack.run_layer(built[L], *inputs[L], tamper=tamperer(L), stream=s))

    with torch.cuda.stream(s):
        for _ in range(warmup):
            one_pass()
    torch.cuda.synchronize()
    gs = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gs, stream=s):
        one_pass()

    def replay_serial():
        with torch.cuda.stream(s):
            gs.replay()

    t_serial = time_passes(replay_serial)
    ok_serial = accepts_ok(results)

    # ---- pipelined ----------------------------------------------------------
    # the four inputs' preparations of every layer spread over the preparation
    # streams (input i on stream i % P), one graph each; each sets its own
    # input's flag, for which that input's masked encode on the online stream
    # waits
    nin = len(stack.INPUTS)
    npre = max(1, args.prep_streams)
    cu_streams = []
    if args.prep_cus and npre == 1:
        # the preparation on compute units [0, prep_cus), the online calls on
        # the rest: neither stream's workgroups wait for the other's units
        ncu = mvk.device_cus()
        if not 0 < args.prep_cus < ncu:
            raise SystemExit(f"--prep-cus must be between 1 and {ncu - 1}")
        cu_streams = [mvk.CUStream(0, args.prep_cus), mvk.CUStream(args.prep_cus, ncu - args.prep_cus)]
        s_preps, s_on = [cu_streams[0].stream], cu_streams[1].stream
    else:
        s_preps, s_on = [torch.cuda.Stream() for _ in range(npre)], torch.cuda.Stream()
    flags = torch.zeros((layers, nin), dtype=torch.int32, device=dev)
    late = torch.zeros((), dtype=torch.int32, device=dev)
    preps = [dict() for _ in range(layers)]
    presults = []

    def prep_pass(k):
        for L in range(layers):
            _, ex, ey = inputs[L]
            if npre == 1:  # the whole layer in one call, one flag
                stack.prepare_layer(built[L], ex, ey, flags[L, 0], out=preps[L], stream=s_preps[0])
                continue
            for i, grp in enumerate(stack.INPUTS):
                if i % npre == k:
                    stack.prepare_input(built[L], grp, ex, ey, preps[L], flag=flags[L, i], stream=s_preps[k])

    def online_pass():
        presults.clear()
        for L in range(layers):
            presults.append(stack.run_layer_prepared(built[L], inputs[L][0], preps[L],
                                                     ready_flag=flags[L, 0] if npre == 1 else
                                                     [flags[L, i] for i in range(nin)],
                                                     timeout_us=200_000, timed_out=late, tamper=tamperer(L),
                                                     stream=s_on))

    for _ in range(warmup):  # also sizes the per-stream workspaces
        for k in range(npre):
            with torch.cuda.stream(s_preps[k]):
                prep_pass(k)
        with torch.cuda.stream(s_on):
            online_pass()
        torch.cuda.synchronize()
    gps = [torch.cuda.CUDAGraph() for _ in range(npre)]
    for k in range(npre):
        with torch.cuda.graph(gps[k], stream=s_preps[k]):
            prep_pass(k)
    go = torch.cuda.CUDAGraph()
    with torch.cuda.graph(go, stream=s_on):
        online_pass()

    def replay_pipelined():
        # a pass's preparation starts after the previous pass's online part
        # (it rewrites the prepared buffers and the flags that part consumes),
        # and is submitted first: streams may share a hardware queue
        for k in range(npre):
            s_preps[k].wait_stream(s_on)
            with torch.cuda.stream(s_preps[k]):
                gps[k].replay()
        with torch.cuda.stream(s_on):
            go.replay()

    late.zero_()
    t_pipe = time_passes(replay_pipelined)
    ok_pipe = accepts_ok(presults) and int(late.item()) == 0
    same = all(bool(torch.equal(a, b)) for sr, pr in zip(results, presults) for name in sr
               for a, b in zip(sr[name], pr[name]))
    del gs, gps, go
    for c in cu_streams:
        c.close()

    # ---- overlapped: the pass on several streams, one graph ----------------
    ov_main = torch.cuda.Stream()
    ov_prep = [torch.cuda.Stream() for _ in range(args.prep_streams)]
    ov_preps = [{name: mvk.Prepared(built[L].keys[name], B, ell) for (name, _, _, _) in stack.PROJECTIONS}
                for L in range(layers)]
    ov_outs = [stack.LayerOutputs.allocate(B, ell) for _ in range(layers)]

    def ov_tamper(L, name, Yhat):
        tamperer(L)(name, Yhat)

    def ov_pass():
        stack.run_pass_overlapped(built, inputs, ov_preps, ov_outs, ov_main, ov_prep, tamper=ov_tamper)

    for _ in range(warmup):  # also sizes every stream's workspace
        with torch.cuda.stream(ov_main):
            ov_pass()
        torch.cuda.synchronize()
    gov = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gov, stream=ov_main):
        ov_pass()

    def replay_overlapped():
        with torch.cuda.stream(ov_main):
            gov.replay()

    t_ov = time_passes(replay_overlapped)
    oresults = [o.as_dict() for o in ov_outs]
    ok_ov = accepts_ok(oresults)
    same_ov = all(bool(torch.equal(a, b)) for sr, orr in zip(results, oresults) for name in sr
                  for a, b in zip(sr[name], orr[name]))
    del gov

    # ---- the pass's server_eval launches alone ------------------------------
    # one server call per layer and input: q, k, v as one grouped launch over
    # their row stack, o alone, up and gate grouped, down alone
    Xs = [{grp: torch.randint(0, P, (B, stack.input_width(grp)), generator=gen, device=dev, dtype=torch.int32)
           for grp in stack.INPUTS} for _ in range(layers)]
    Ys = {name: torch.empty((B, m), dtype=torch.int32, device=dev) for (name, m, _, _) in stack.PROJECTIONS}
    calls = [(L, grp) for L in range(layers) for grp in stack.INPUTS]

    def launches(items):
        for (L, grp) in items:
            stack.evaluate_stage(built[L], grp, Xs[L][grp], outs=Ys, stream=s)

    def alg_bytes(grp):
        return sum(m * n + 4 * n * B + 4 * m * B for (name, m, n, g) in stack.PROJECTIONS if g == grp)

    pass_s = graph_mean_seconds(s, lambda k: launches(calls), steps, args.warm_seconds)
    alg_pass = sum(alg_bytes(grp) for (_, grp) in calls)
    per_shape = {}
    for grp in stack.INPUTS:
        items = [c for c in calls if c[1] == grp]
        t = graph_mean_seconds(s, lambda k, it=items: launches(it), max(2, steps // 4), args.warm_seconds)
        t_launch = t / len(items)
        names = stack.stage(grp)
        m, n = next((m, n) for (nm, m, n, _) in stack.PROJECTIONS if nm == names[0])
        label = f"{','.join(names)}: {len(names)}x{m}x{n}" if len(names) > 1 else f"{names[0]}: {m}x{n}"
        per_shape[label] = {"launches_per_pass": len(items), "mean_launch_us": 1e6 * t_launch,
                            "alg_bytes_per_launch": alg_bytes(grp), "gbps": alg_bytes(grp) / t_launch / 1e9,
                            "frac": alg_bytes(grp) / t_launch / 1e9 / HBM_PEAK_GBS}
    every = [(L, name, grp) for (L, grp) in calls for name in stack.stage(grp)]
    read_s = read_floor([built[L].W[name].data for (L, name, _) in every], len(every), args)
    achieved = alg_pass / pass_s / 1e9
    macs = stack.macs_per_layer(B) * layers
    elapsed = {"pipelined": t_pipe, "serial": t_serial, "overlapped": t_ov}[args.stack_mode]
    res = {"metric": METRIC, "value": macs / elapsed, "unit": "modMAC/s", "n_gpus": 1, "steps": steps,
           "warmup": warmup, "ms_per_step": 1e3 * elapsed, "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": DTYPE, "data": "synthetic",
           "config": {"workload": f"stack32: {layers} layers x (q,k,v,o 4096x4096; up,gate 11008x4096; "
                                  f"down 4096x11008) int8-valued W in F_p (p=2^31-1), B={B} query columns per "
                                  f"projection, RAA r={r}, t_x={tx}, t_y={ty}, ell={ell}; step = one pass (per layer "
                                  "4 encodes, 7 server_evals, 7 decode_verifies) with one response in 1000 "
                                  "tampered and rejected",
                      "global_batch": B, "launch": "hip_graph", "mode": args.stack_mode, "weights": "packed",
                      "prep_cus": args.prep_cus if args.stack_mode == "pipelined" else None},
           "ms_per_step_overlapped": 1e3 * t_ov, "ms_per_step_pipelined": 1e3 * t_pipe,
           "ms_per_step_serial": 1e3 * t_serial,
           "modmac_per_pass": macs,
           "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": achieved / HBM_PEAK_GBS, "traffic": measured_traffic("stack32", "packed"),
                        "kernel": f"server_eval ({args.path}), the {len(calls)} server calls of a pass back to "
                                  f"back ({len(every)} products: q,k,v and up,gate grouped over their shared input)",
                        "alg_bytes_per_launch": alg_pass / len(calls), "alg_bytes_per_pass": alg_pass,
                        "launches_per_pass": len(calls), "mean_launch_us": 1e6 * pass_s / len(calls),
                        "server_ms_per_pass": 1e3 * pass_s, "per_shape": per_shape,
                        "read_floor": {"ms_per_pass": 1e3 * read_s * len(every),
                                       "gbps": alg_pass / (read_s * len(every)) / 1e9,
                                       "frac": read_s * len(every) / pass_s,
                                       "what": "a streaming read of the same W buffers, one launch per matrix"}},
           "server_eval": {"modmac_per_s": macs / pass_s, "gb_per_s": achieved},
           "preprocess": preprocess_record(stack, r, pre_ms),
           "tampered_per_pass": sum(len(v) for v in plan.values()),
           "all_expected_verdicts": ok_serial and ok_pipe and ok_ov, "pipelined_matches_serial": same,
           "overlapped_matches_serial": same_ov, "setup_s": t_setup}
    del built, inputs, results, presults, preps, Xs, Ys, oresults, ov_outs, ov_preps
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline_stack(cpu_seconds)
    res["_ok"] = ok_serial and ok_pipe and ok_ov and same and same_ov
    return res


def preprocess_record(stack, r, ms):
    """Preprocess of one stack layer (keygen of the seven projections: P^T and
    Q by the batched RAA encoding, then packing W), HIP events per layer.  The
    algorithmic bytes are W read twice (keygen, packing), P^T and Q written
    and the packed W written; frac is against the HBM peak."""
    import numpy as np

    alg = sum(2 * m * n + 4 * r * n * m + 4 * r * m * n + m * n for (_, m, n, _) in stack.PROJECTIONS)
    t = float(np.mean(ms)) if ms else float("nan")
    return {"ms_per_layer": t, "layers_timed": len(ms), "alg_bytes_per_layer": alg,
            "gb_per_s": alg / (1e-3 * t) / 1e9, "frac": alg / (1e-3 * t) / 1e9 / HBM_PEAK_GBS}


def cpu_baseline_config(cfg, seconds):
    """The oracle's whole step (encode, server_eval, verify, decode) on the
    workload's shapes, threaded over row blocks on every core of this host,
    timed over repeated steps for about `seconds` (preprocessing untimed)."""
    import oracle
    import synth

    m, n, B, r, tx, ty, ell = (cfg[k] for k in ("m", "n", "B", "r", "tx", "ty", "ell"))
    cid = cfg["cid"]
    T = oracle.threads()
    cx = synth.raa_code(synth.seed_for(cid, synth.PURPOSE_CX), n, r)
    cy = synth.raa_code(synth.seed_for(cid, synth.PURPOSE_CY), m, r)
    W = synth.weights(synth.seed_for(cid, synth.PURPOSE_W, 5), m, n)
    PT, Q = oracle.keygen(W, cx, cy, nthreads=T)  # preprocessing, untimed
    steps, el = 0, 0.0
    while True:
        X = synth.field_uniform(synth.seed_for(cid, synth.PURPOSE_X, 100 + steps), (B, n))
        exi, exv = synth.sparse(synth.seed_for(cid, synth.PURPOSE_NOISE, 100 + steps), B, cx["N"], tx)
        eyi, eyv = synth.sparse(synth.seed_for(cid, synth.PURPOSE_CHAL, 100 + steps), ell, cy["N"], ty)
        t0 = time.perf_counter()
        Xh = oracle.encode(cx, X, exi, exv)
        Yh = oracle.server_eval(W, Xh, nthreads=T)
        acc, _, _ = oracle.verify(cy, Q, Xh, Yh, eyi, eyv)
        oracle.decode(PT, Yh, exi, exv, nthreads=T)
        el += time.perf_counter() - t0
        assert acc.all()
        steps += 1
        if el >= seconds or steps >= 10000:
            break
    return {"value": m * n * B * steps / el, "unit": "modMAC/s", "cores": T, "kind": "oracle",
            "host_cpu": host_cpu(),
            "sample": f"{steps} whole steps (encode+server_eval+verify+decode) of the same shapes, one W, "
                      f"{el:.1f} s of oracle time (input drawing and preprocessing excluded); plain C, '%' per "
                      f"field op, server product and decryption split over {T} threads by row blocks"}


def cpu_baseline_stack(seconds):
    """The oracle on one layer of the stack (4 encodes, 7 server products, 7
    verifications and decryptions), threaded over row blocks on every core,
    repeated for about `seconds`; scaled to mod-MAC/s like the GPU pass."""
    import oracle
    import paper_2609_10264_amd.stack as stack
    import synth

    cfg = synth.STACK
    B, r, tx, ty, ell, cid = (cfg[k] for k in ("B", "r", "tx", "ty", "ell", "cid"))
    T = oracle.threads()
    cxs = {n: synth.raa_code(synth.seed_for(cid, synth.PURPOSE_CX, sub=n), n, r)
           for n in {n for (_, _, n, _) in stack.PROJECTIONS}}
    cys = {m: synth.raa_code(synth.seed_for(cid, synth.PURPOSE_CY, sub=m), m, r)
           for m in {m for (_, m, _, _) in stack.PROJECTIONS}}
    Ws, keys = {}, {}
    for i, (name, m, n, _) in enumerate(stack.PROJECTIONS):
        Ws[name] = synth.weights(synth.seed_for(cid, synth.PURPOSE_W, 900 + i), m, n)
        keys[name] = oracle.keygen(Ws[name], cxs[n], cys[m], nthreads=T)  # preprocessing, untimed
    steps, el = 0, 0.0
    while True:
        X, ex = {}, {}
        for j, grp in enumerate(stack.INPUTS):
            n = stack.input_width(grp)
            X[grp] = synth.field_uniform(synth.seed_for(cid, synth.PURPOSE_X, 900 + 10 * steps + j), (B, n))
            ex[grp] = synth.sparse(synth.seed_for(cid, synth.PURPOSE_NOISE, 900 + 10 * steps + j), B, r * n, tx)
        ey = {name: synth.sparse(synth.seed_for(cid, synth.PURPOSE_CHAL, 900 + 10 * steps + i), ell, r * m, ty)
              for i, (name, m, _, _) in enumerate(stack.PROJECTIONS)}
        t0 = time.perf_counter()
        Xh = {grp: oracle.encode(cxs[stack.input_width(grp)], X[grp], *ex[grp]) for grp in stack.INPUTS}
        ok = True
        for name, m, n, grp in stack.PROJECTIONS:
            PT, Q = keys[name]
            Yh = oracle.server_eval(Ws[name], Xh[grp], nthreads=T)
            acc, _, _ = oracle.verify(cys[m], Q, Xh[grp], Yh, *ey[name])
            oracle.decode(PT, Yh, *ex[grp], nthreads=T)
            ok = ok and bool(acc.all())
        el += time.perf_counter() - t0
        assert ok
        steps += 1
        if el >= seconds:
            break
    macs = stack.macs_per_layer(B)
    return {"value": macs * steps / el, "unit": "modMAC/s", "cores": T, "kind": "oracle", "host_cpu": host_cpu(),
            "sample": f"{steps} steps of one layer of the stack (4 encodes, 7 server products, 7 verifications "
                      f"and decryptions; {macs / 1e9:.2f} G mod-MACs each), {el:.1f} s of oracle time (input drawing "
                      f"and preprocessing excluded); plain C, '%' per field op, server products and decryptions "
                      f"split over {T} threads by row blocks"}


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
        kg_bytes = m * n + 4 * r * n * m + 4 * r * m * n  # W read, P^T and Q written
        kg_s = 1e-3 * float(np.mean(kg_ms))
        rows.append({"n": n, "t_x": tx, "w_pool": pool, "keygen_ms": float(np.mean(kg_ms)),
                     "keygen_gb_per_s": kg_bytes / kg_s / 1e9, "keygen_hbm_frac": kg_bytes / kg_s / 1e9 / HBM_PEAK_GBS,
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
        T = oracle.threads()
        rows_s = 64 * T
        Wh = synth.weights(synth.seed_for(cid, synth.PURPOSE_W, n), rows_s, n)
        Xq = synth.field_uniform(synth.seed_for(cid, synth.PURPOSE_X, n), (1, n), p=p)
        reps, el = 0, 0.0
        while el < min(args.cpu_seconds, 5.0):
            t0 = time.perf_counter()
            oracle.server_eval(Wh, Xq, p=p, nthreads=T)
            el += time.perf_counter() - t0
            reps += 1
        res["cpu_baseline"] = {"value": rows_s * n * reps / el, "unit": "modMAC/s", "cores": T, "kind": "oracle",
                               "host_cpu": host_cpu(),
                               "sample": f"{reps} oracle server products of {rows_s} rows x {n} over BabyBear, "
                                         f"{el:.1f} s; plain C, '%' per field op, rows split over {T} threads"}
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


if __name__ == "__main__":
    main()
