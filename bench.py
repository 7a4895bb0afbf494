#!/usr/bin/env python3
"""Benchmark of the resonant mixing hot path on one MI355X.

One step = one prefill forward pass of the long-context workload (B=4, L=32768,
D=256, M=8, bf16 drive and output, fp32 accumulation, terminal state written):
parameter tables, chunk products, cross-tile carry, correction and store.  The
timed region holds exactly K steps with the inputs already resident in HBM;
three input/output buffer sets rotate so that the working set (3 x 134 MB)
exceeds the 256 MB Infinity Cache.  The JSON line also carries

  decode    steps/s of the decode workload (B=64, D=256, M=8, state from a
            1024-step prompt), eager (one C call per step from Python) and
            replayed from a captured HIP graph of the same calls;
  train     one forward + backward of a training layer (B=8, L=8192, D=256, M=8,
            bf16), as time per layer;
  roofline  the dominant kernel (the single-pass streaming forward kernel) against the HBM
            peak: algorithmic bytes (2 B read + 2 B written per token-channel)
            per launch over its average launch time, measured with HIP events
            recorded around that kernel alone;
  cpu_baseline  the float64 CPU oracle (sequential recurrence) on the host.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
COPY_BYTES = 256 << 20  # calibration copy of the counter run
METRIC = "prefill mix tokens·ch/s + decode steps/s at L=32K; % of HBM peak"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_fwd_stream_prefill_B4_L32768_D256_M8.json")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def counter_traffic(per_launch_tokens: int):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it was
    taken on the current kernel sources; else None."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    with open(TRAFFIC_FILE) as f:
        t = json.load(f)
    from paper_2607_05583_amd.profiling import source_hash
    if t.get("source_hash") != source_hash():
        return None
    return t.get("bytes_per_launch")


def _oracle_passes(args):
    """Worker of the multi-process CPU leg: whole passes of the oracle recurrence
    over one channel slice until min_s seconds of work; returns (passes, seconds)."""
    x, prm, min_s = args
    os.environ.setdefault("OMP_NUM_THREADS", "1")
    import oracle as O
    passes, t0 = 0, time.perf_counter()
    while True:
        O.mix_recurrence(x, *prm)
        passes += 1
        dt = time.perf_counter() - t0
        if dt >= min_s:
            return passes, dt


def cpu_baseline(cfg, min_s=10.0):
    """The oracle's sequential recurrence on the prefill workload, timed on the
    host: one thread, then the channels split over one process per available
    core (the recurrence of one channel is independent of the others)."""
    import multiprocessing as mp
    from concurrent.futures import ProcessPoolExecutor

    import oracle as O
    import workloads as W
    inp = W.fwd_inputs(cfg)
    x = W.act_to_f32(inp["x"], cfg.act).astype(np.float64)
    prm = [inp[k] for k in ("gamma", "omega", "amp", "phase")]
    # one thread: whole passes over the workload until min_s seconds of CPU work
    passes, t0 = 0, time.perf_counter()
    while True:
        O.mix_recurrence(x, *prm)
        passes += 1
        dt = time.perf_counter() - t0
        if dt >= min_s or passes >= 30:
            break
    n1 = cfg.B * cfg.L * cfg.D * passes
    single = {"value": n1 / dt, "unit": "tokens*ch/s", "cores": 1, "kind": "oracle",
              "sample": f"{passes} passes over the whole prefill workload B={cfg.B} L={cfg.L} D={cfg.D} "
                        f"M={cfg.M}: float64 numpy recurrence vectorised over (b, d, m), one host thread, "
                        f"{dt:.1f} s in all"}
    # all cores: the channels split into one slice per process (spawned before
    # this process touches the GPU), each running whole passes for min_s seconds
    cores = len(os.sched_getaffinity(0))
    nproc = max(1, min(cores, 16, cfg.D))
    bounds = np.linspace(0, cfg.D, nproc + 1).astype(int)
    tasks = [(np.ascontiguousarray(x[:, :, a:b]), [v[a:b] for v in prm], min_s)
             for a, b in zip(bounds[:-1], bounds[1:])]
    t0 = time.perf_counter()
    with ProcessPoolExecutor(max_workers=nproc, mp_context=mp.get_context("spawn")) as ex:
        res = list(ex.map(_oracle_passes, tasks))
    wall = time.perf_counter() - t0
    done = sum(p * cfg.B * cfg.L * (b - a) for (p, _), a, b in zip(res, bounds[:-1], bounds[1:]))
    longest = max(t for _, t in res)
    return {"value": done / longest, "unit": "tokens*ch/s", "cores": nproc, "kind": "oracle",
            "sample": f"the prefill workload B={cfg.B} L={cfg.L} D={cfg.D} M={cfg.M} with its channels split "
                      f"over {nproc} processes ({cores} cores available), each running whole float64 passes of "
                      f"the oracle recurrence over its {cfg.D // nproc}-{-(-cfg.D // nproc)} channels for at "
                      f"least {min_s:.0f} s ({wall:.1f} s wall with start-up); throughput = channel-steps done "
                      f"over the longest worker time",
            "single_thread": single}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--decode-steps", type=int, default=32768)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--counters", nargs="?", const="fwd", choices=("fwd", "bwd", "decode", "block", "block_bwd"),
                    help="short run for rocprofv3 --pmc: one runtime buffer copy of COPY_BYTES "
                         "(the counter calibration), then --steps launches of one workload: the "
                         "prefill forward on rotating buffers (fwd, the default), one training "
                         "layer's forward and backward (bwd), or graph decode replays of 64 steps "
                         "(decode); prints one JSON line and skips everything else")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: this build runs the operator on a single "
              f"MI355X (got --gpus {args.gpus}); sharding across GPUs is not part of it.",
              file=sys.stderr)
        sys.exit(2)

    import workloads as W
    cpu = None
    if not args.no_cpu and not args.counters:
        log("cpu baseline (oracle recurrence, one thread and all cores) ...")
        cpu = cpu_baseline(W.CONFIGS[3])

    import torch
    from paper_2607_05583_amd import _lib, ops
    from paper_2607_05583_amd._lib import RES_OP_FWD

    assert torch.cuda.is_available(), "bench.py needs a HIP device"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    lib = _lib.lib()

    # ---------------- prefill (the timed step) ----------------
    cfg = W.CONFIGS[3]
    log(f"prefill workload {cfg.name}")
    inp = W.fwd_inputs(cfg)
    prm = [torch.from_numpy(inp[k]).to(dev) for k in ("gamma", "omega", "amp", "phase")]
    x0 = torch.from_numpy(inp["x"].view(np.int16)).view(torch.bfloat16).to(dev)
    NSET = 3
    xs = [x0] + [x0.roll(shifts=i * 997, dims=1).contiguous() for i in range(1, NSET)]
    ys = [torch.empty_like(x0) for _ in range(NSET)]
    hs = [torch.empty((cfg.B, cfg.D, cfg.M, 2), dtype=torch.float32, device=dev) for _ in range(NSET)]
    B, L, D, M = cfg.B, cfg.L, cfg.D, cfg.M
    wsn = ops.workspace_bytes(RES_OP_FWD, torch.bfloat16, B, L, D, M)
    ws = torch.zeros(wsn, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    import ctypes
    sp = ctypes.c_void_p(stream.cuda_stream)
    P = [ctypes.c_void_p(p.data_ptr()) for p in prm]

    def fwd(i, ev=None):
        if ev is not None:
            _lib.check(lib.resonator_set_kernel_timer(ctypes.c_void_p(ev[0].cuda_event),
                                                      ctypes.c_void_p(ev[1].cuda_event)))
        _lib.check(lib.resonator_mix_fwd(
            ctypes.c_void_p(xs[i].data_ptr()), _lib.RES_BF16, ctypes.c_void_p(ys[i].data_ptr()),
            _lib.RES_BF16, B, L, D, M, *P, None, ctypes.c_void_p(hs[i].data_ptr()),
            ctypes.c_void_p(ws.data_ptr()), wsn, sp))

    if args.counters:
        src = torch.empty(COPY_BYTES, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        name = cfg.name
        if args.counters == "fwd":
            for i in range(args.steps):
                fwd(i % NSET)
        elif args.counters == "bwd":
            c5 = W.CONFIGS[5]
            name = c5.name + " layer 0"
            li = W.train_layer_inputs(c5, 0)
            tprm = [torch.from_numpy(li[k]).to(dev) for k in ("gamma", "omega", "amp", "phase")]
            tx = torch.from_numpy(li["x"].view(np.int16)).view(torch.bfloat16).to(dev)
            tdy = torch.from_numpy(li["dy"].view(np.int16)).view(torch.bfloat16).to(dev)
            TB, TL, TD, TM = tx.shape[0], tx.shape[1], tx.shape[2], tprm[0].shape[1]
            tfws = ops.forward_workspace(torch.bfloat16, TB, TL, TD, TM, dev)
            tbws = torch.empty(max(ops.workspace_bytes(ops.RES_OP_BWD, torch.bfloat16, TB, TL, TD, TM), 256),
                               dtype=torch.uint8, device=dev)
            for _ in range(args.steps):
                ops.resonator_mix_fwd(tx, *tprm, ws=tfws)
                ops.resonator_mix_bwd(tx, tdy, *tprm, ws=tbws)
        elif args.counters == "block":
            name = "mixer block forward B4 L32768 d256 bf16 (H8 x dh32, K4, 8 groups, M8)"
            pb_ = W.block_inputs(13, 4, 32768, 256, 8, 4, 8, 8, "bf16")
            bt = {k: torch.from_numpy(pb_[k].view(np.int16)).view(torch.bfloat16).to(dev) for k in ("x", "Wu", "Wg", "Wo")}
            bp = [torch.from_numpy(pb_[k]).to(dev) for k in ("gamma", "omega", "amp", "phase", "Ct", "w", "s")]
            for _ in range(args.steps):
                ops.resonator_block_fwd(bt["x"], bt["Wu"], bt["Wg"], bt["Wo"], *bp[:4], bp[4], 0.5, bp[5], bp[6], 8)
        elif args.counters == "block_bwd":
            name = "mixer block backward B4 L32768 d256 bf16 (H8 x dh32, K4, 8 groups, M8), recomputing the forward"
            pb_ = W.block_inputs(13, 4, 32768, 256, 8, 4, 8, 8, "bf16")
            bt = {k: torch.from_numpy(pb_[k].view(np.int16)).view(torch.bfloat16).to(dev) for k in ("x", "Wu", "Wg", "Wo")}
            bp = [torch.from_numpy(pb_[k]).to(dev) for k in ("gamma", "omega", "amp", "phase", "Ct", "w", "s")]
            dob = torch.randn_like(bt["x"], dtype=torch.float32).to(torch.bfloat16)
            for _ in range(args.steps):
                ops.resonator_block_bwd(bt["x"], bt["Wu"], bt["Wg"], bt["Wo"], *bp[:4], bp[4], 0.5, bp[5], bp[6], 8, dob)
        else:
            c4 = W.CONFIGS[4]
            name = c4.name + " graph replays of 64 steps"
            di = W.DecodeInputs(c4)
            dprm = [torch.from_numpy(di.params[k]).to(dev) for k in ("gamma", "omega", "amp", "phase")]
            prompt = torch.from_numpy(di.prompt.view(np.int16)).view(torch.bfloat16).to(dev)
            state = ops.resonator_state_init(prompt, *dprm)
            g = ops.DecodeGraph(*dprm, state, 64, x_dtype=torch.bfloat16)
            g.x.copy_(torch.randn(g.x.shape, device=dev).to(torch.bfloat16))
            for _ in range(args.steps):
                g.replay()
        torch.cuda.synchronize()
        print(json.dumps({"counters_run": True, "copy_bytes": COPY_BYTES, "launches": args.steps,
                          "counters": args.counters, "workload": name}), flush=True)
        return

    for i in range(args.warmup):
        fwd(i % NSET)
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for a, b in evs:  # torch creates events lazily: record once so the handles exist
        a.record(stream)
        b.record(stream)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # The step time comes from K steps as a caller runs them.  Timing events
    # around each kernel (hipExtLaunchKernelGGL with start and stop events) add
    # about 6 us of dispatch gap per launch, so the kernel's own duration comes
    # from a second run of K steps with those events.
    torch.cuda.synchronize()
    t_wall0 = time.perf_counter()
    start.record(stream)
    for i in range(args.steps):
        fwd(i % NSET)
    stop.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall0
    ms_total = start.elapsed_time(stop)
    ms_step = ms_total / args.steps
    start.record(stream)
    for i in range(args.steps):
        fwd(i % NSET, evs[i])
    stop.record(stream)
    torch.cuda.synchronize()
    ms_step_ev = start.elapsed_time(stop) / args.steps
    k_ms = [a.elapsed_time(b) for a, b in evs]
    k_avg_ms = float(np.mean(k_ms))
    n_tok = B * L * D
    value = n_tok / (ms_step * 1e-3)
    alg_bytes = n_tok * 4
    achieved = alg_bytes / (k_avg_ms * 1e-3) / 1e9
    log(f"prefill: {ms_step * 1e3:.1f} us/step (events), forward kernel {k_avg_ms * 1e3:.1f} us "
        f"({ms_step_ev * 1e3:.1f} us/step with per-kernel events), wall {t_wall / args.steps * 1e6:.1f} us/step")

    # ---------------- prefill across lengths (1K .. 32K tokens) ----------------
    # B4 D256 M8 bf16 as the prefill config, L from 1K to 32K; the step and the
    # forward kernel alone, with its share of the HBM roofline
    sweep = []
    for Ls in (1024, 2048, 4096, 8192, 16384, 32768):
        xl = torch.randn((B, Ls, D), generator=torch.Generator(device=dev).manual_seed(Ls), device=dev,
                         dtype=torch.float32).to(torch.bfloat16)
        yl = torch.empty_like(xl)
        hl = torch.empty((B, D, M, 2), dtype=torch.float32, device=dev)
        wn = ops.workspace_bytes(RES_OP_FWD, torch.bfloat16, B, Ls, D, M)
        wl = torch.zeros(wn, dtype=torch.uint8, device=dev)
        ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))

        def fwd_l(timed):
            if timed:
                _lib.check(lib.resonator_set_kernel_timer(ctypes.c_void_p(ev[0].cuda_event),
                                                          ctypes.c_void_p(ev[1].cuda_event)))
            _lib.check(lib.resonator_mix_fwd(
                ctypes.c_void_p(xl.data_ptr()), _lib.RES_BF16, ctypes.c_void_p(yl.data_ptr()), _lib.RES_BF16,
                B, Ls, D, M, *P, None, ctypes.c_void_p(hl.data_ptr()), ctypes.c_void_p(wl.data_ptr()), wn, sp))

        ev[0].record(stream)
        ev[1].record(stream)
        for _ in range(3):
            fwd_l(False)
        torch.cuda.synchronize()
        reps = max(5, min(200, (1 << 22) // Ls))
        start.record(stream)
        for _ in range(reps):
            fwd_l(False)
        stop.record(stream)
        torch.cuda.synchronize()
        st_us = start.elapsed_time(stop) * 1e3 / reps
        kus = []
        for _ in range(5):
            fwd_l(True)
            torch.cuda.synchronize()
            kus.append(ev[0].elapsed_time(ev[1]) * 1e3)
        k_us = float(np.median(kus))
        gbs = B * Ls * D * 4 / (k_us * 1e-6) / 1e9
        sweep.append({"L": Ls, "B": B, "step_us": st_us, "tokens_ch_per_s": B * Ls * D / (st_us * 1e-6),
                      "fwd_kernel_us": k_us, "fwd_kernel_GBs": gbs, "frac_of_hbm_peak": gbs / HBM_PEAK_GBS})
        log(f"prefill L={Ls}: step {st_us:.1f} us, forward kernel {k_us:.1f} us ({gbs:.0f} GB/s)")
        del xl, yl, wl

    # ---------------- measured copy bandwidth (the practical HBM ceiling) ----------------
    # a device-to-device copy of 1 GiB (read + write), well beyond the Infinity Cache
    csrc = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(1)
    cdst = torch.empty_like(csrc)
    for _ in range(2):
        cdst.copy_(csrc)
    torch.cuda.synchronize()
    creps = 10
    start.record(stream)
    for _ in range(creps):
        cdst.copy_(csrc)
    stop.record(stream)
    torch.cuda.synchronize()
    copy_gbs = 2 * csrc.numel() / (start.elapsed_time(stop) * 1e-3 / creps) / 1e9
    del csrc, cdst
    log(f"device copy: {copy_gbs:.0f} GB/s (read + write)")

    # ---------------- configs 1 and 2 (float32 forward) ----------------
    fcfg = []
    for k in (1, 2):
        ck = W.CONFIGS[k]
        ik = W.fwd_inputs(ck)
        xk_ = torch.from_numpy(ik["x"]).to(dev)
        yk_ = torch.empty_like(xk_)
        pk_ = [torch.from_numpy(ik[n]).to(dev) for n in ("gamma", "omega", "amp", "phase")]
        wn_ = ops.workspace_bytes(RES_OP_FWD, torch.float32, ck.B, ck.L, ck.D, ck.M)
        wk_ = torch.zeros(wn_, dtype=torch.uint8, device=dev)
        PK = [ctypes.c_void_p(p.data_ptr()) for p in pk_]
        evk = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))

        def fwd_k(timed):
            if timed:
                _lib.check(lib.resonator_set_kernel_timer(ctypes.c_void_p(evk[0].cuda_event),
                                                          ctypes.c_void_p(evk[1].cuda_event)))
            _lib.check(lib.resonator_mix_fwd(
                ctypes.c_void_p(xk_.data_ptr()), _lib.RES_F32, ctypes.c_void_p(yk_.data_ptr()), _lib.RES_F32,
                ck.B, ck.L, ck.D, ck.M, *PK, None, None, ctypes.c_void_p(wk_.data_ptr()), wn_, sp))

        evk[0].record(stream)
        evk[1].record(stream)
        for _ in range(3):
            fwd_k(False)
        torch.cuda.synchronize()
        reps = 50
        start.record(stream)
        for _ in range(reps):
            fwd_k(False)
        stop.record(stream)
        torch.cuda.synchronize()
        st_us = start.elapsed_time(stop) * 1e3 / reps
        kus = []
        for _ in range(10):
            fwd_k(True)
            torch.cuda.synchronize()
            kus.append(evk[0].elapsed_time(evk[1]) * 1e3)
        k_us = float(np.median(kus))
        ntk = ck.B * ck.L * ck.D
        gbs = ntk * 8 / (k_us * 1e-6) / 1e9
        fcfg.append({"config": k, "workload": ck.name, "step_us": st_us, "tokens_ch_per_s": ntk / (st_us * 1e-6),
                     "kernel_us": k_us, "kernel_alg_GBs": gbs, "frac_of_hbm_peak": gbs / HBM_PEAK_GBS})
        log(f"config {k} ({ck.name}): step {st_us:.1f} us, kernel {k_us:.1f} us ({gbs:.0f} GB/s)")
        del xk_, yk_, wk_

    # ---------------- decode ----------------
    c4 = W.CONFIGS[4]
    log(f"decode workload {c4.name}")
    di = W.DecodeInputs(c4)
    dprm = [torch.from_numpy(di.params[k]).to(dev) for k in ("gamma", "omega", "amp", "phase")]
    prompt = torch.from_numpy(di.prompt.view(np.int16)).view(torch.bfloat16).to(dev)
    state = ops.resonator_state_init(prompt, *dprm)
    nsteps = args.decode_steps
    chunk = 4096
    xdec = torch.from_numpy(di.steps(min(chunk, nsteps)).view(np.int16)).view(torch.bfloat16).to(dev)
    ydec = torch.empty_like(xdec)
    DP = [ctypes.c_void_p(p.data_ptr()) for p in dprm]
    sptr = ctypes.c_void_p(state.data_ptr())
    Bd, Dd, Md = c4.B, c4.D, c4.M
    xptr = [ctypes.c_void_p(xdec[j].data_ptr()) for j in range(xdec.shape[0])]
    yptr = [ctypes.c_void_p(ydec[j].data_ptr()) for j in range(xdec.shape[0])]

    def dstep(j):
        _lib.check(lib.resonator_decode_step(xptr[j], _lib.RES_BF16, yptr[j], _lib.RES_BF16, Bd, Dd,
                                             Md, *DP, sptr, sp))

    for j in range(64):
        dstep(j)
    torch.cuda.synchronize()
    d0, d1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    d0.record(stream)
    for s in range(nsteps):
        dstep(s % xdec.shape[0])
    d1.record(stream)
    torch.cuda.synchronize()
    dec_eager_us = d0.elapsed_time(d1) * 1e3 / nsteps
    # graph replay of the same calls (kernel launches only; no allocation, no memset)
    G = min(512, int(xdec.shape[0]))
    dgraph = ops.DecodeGraph(*dprm, state, G, x_dtype=torch.bfloat16)
    dgraph.x.copy_(xdec[:G])
    torch.cuda.synchronize()
    dgraph.replay()
    torch.cuda.synchronize()
    g = dgraph.graph
    reps = max(1, nsteps // G)
    d0.record(stream)
    for _ in range(reps):
        g.replay()
    d1.record(stream)
    torch.cuda.synchronize()
    dec_graph_us = d0.elapsed_time(d1) * 1e3 / (reps * G)
    # launch floor of a replayed graph: G launches of a one-element kernel
    tiny = torch.zeros(1, dtype=torch.float32, device=dev)
    fgraph = torch.cuda.CUDAGraph()
    fcap = torch.cuda.Stream(dev)
    fcap.wait_stream(stream)
    with torch.cuda.stream(fcap), torch.cuda.graph(fgraph, stream=fcap):
        for _ in range(G):
            tiny.add_(1.0)
    stream.wait_stream(fcap)
    fgraph.replay()
    torch.cuda.synchronize()
    d0.record(stream)
    for _ in range(reps):
        fgraph.replay()
    d1.record(stream)
    torch.cuda.synchronize()
    floor_us = d0.elapsed_time(d1) * 1e3 / (reps * G)
    del fgraph
    dec_bytes = Bd * Dd * (Md * 16 + 2 + 2)
    log(f"decode: eager {dec_eager_us:.2f} us/step, graph {dec_graph_us:.2f} us/step "
        f"(replayed one-element launches: {floor_us:.2f} us each)")
    # several steps per launch, for drives known in advance: 8 drafted tokens to
    # verify per launch, and a long run of known drives in one launch
    xbn = xdec.permute(1, 0, 2).contiguous()  # [B, N, D]
    ybn = torch.empty_like(xbn)
    xk = xbn[:, :8].contiguous()
    yk = torch.empty_like(xk)
    st_ms = state.clone()
    msp = ctypes.c_void_p(st_ms.data_ptr())

    def msteps(xt, yt):
        _lib.check(lib.resonator_decode_steps(ctypes.c_void_p(xt.data_ptr()), _lib.RES_BF16,
                                              ctypes.c_void_p(yt.data_ptr()), _lib.RES_BF16, Bd, xt.shape[1],
                                              Dd, Md, *DP, msp, sp))

    for _ in range(5):
        msteps(xk, yk)
    msteps(xbn, ybn)
    torch.cuda.synchronize()
    nk = 2000
    d0.record(stream)
    for _ in range(nk):
        msteps(xk, yk)
    d1.record(stream)
    torch.cuda.synchronize()
    k8_us = d0.elapsed_time(d1) * 1e3 / nk
    nl = 5
    d0.record(stream)
    for _ in range(nl):
        msteps(xbn, ybn)
    d1.record(stream)
    torch.cuda.synchronize()
    long_us = d0.elapsed_time(d1) * 1e3 / (nl * xbn.shape[1])
    log(f"decode, several steps per launch: 8 steps {k8_us:.2f} us per launch ({k8_us / 8:.2f} us/step), "
        f"{xbn.shape[1]} steps {long_us:.3f} us/step")
    del xbn, ybn, st_ms

    # ---------------- training layer (fwd + bwd) ----------------
    c5 = W.CONFIGS[5]
    li = W.train_layer_inputs(c5, 0)
    tprm = [torch.from_numpy(li[k]).to(dev) for k in ("gamma", "omega", "amp", "phase")]
    tx = torch.from_numpy(li["x"].view(np.int16)).view(torch.bfloat16).to(dev)
    tdy = torch.from_numpy(li["dy"].view(np.int16)).view(torch.bfloat16).to(dev)
    # workspaces allocated once and reused by every call, as in a training loop
    TB, TL, TD, TM = tx.shape[0], tx.shape[1], tx.shape[2], tprm[0].shape[1]
    tfws = ops.forward_workspace(torch.bfloat16, TB, TL, TD, TM, dev)
    tbws = torch.empty(max(ops.workspace_bytes(ops.RES_OP_BWD, torch.bfloat16, TB, TL, TD, TM), 256),
                       dtype=torch.uint8, device=dev)
    for _ in range(3):
        ops.resonator_mix_fwd(tx, *tprm, ws=tfws)
        ops.resonator_mix_bwd(tx, tdy, *tprm, ws=tbws)
    torch.cuda.synchronize()
    nt = 10
    t0e, t1e, t2e, t3e = (torch.cuda.Event(enable_timing=True) for _ in range(4))
    t0e.record(stream)
    for _ in range(nt):
        ops.resonator_mix_fwd(tx, *tprm, ws=tfws)
    t1e.record(stream)
    for _ in range(nt):
        ops.resonator_mix_bwd(tx, tdy, *tprm, ws=tbws)
    t2e.record(stream)
    torch.cuda.synchronize()
    tr_fwd_us = t0e.elapsed_time(t1e) * 1e3 / nt
    tr_bwd_us = t1e.elapsed_time(t2e) * 1e3 / nt
    log(f"train layer: fwd {tr_fwd_us:.1f} us, bwd {tr_bwd_us:.1f} us")

    # ---------------- mixer epilogue (head coupling, gate, local path) ----------------
    eB, eL, eH, edh, eK = cfg.B, cfg.L, 8, cfg.D // 8, 4
    ep = W.epilogue_inputs(11, eB, eL, eH, edh, eK, "bf16")
    et = {k: torch.from_numpy(ep[k].view(np.int16)).view(torch.bfloat16).to(dev) for k in ("y", "gate", "v", "dz")}
    eCt, ew, es = (torch.from_numpy(ep[k]).to(dev) for k in ("Ct", "w", "s"))
    del ep
    efwd = lambda: ops.resonator_epilogue_fwd(et["y"], et["gate"], et["v"], eCt, 0.5, ew, es, eH)
    ebwd = lambda: ops.resonator_epilogue_bwd(et["y"], et["gate"], et["v"], et["dz"], eCt, 0.5, ew, es, eH)
    for _ in range(3):
        efwd(), ebwd()
    torch.cuda.synchronize()
    t0e.record(stream)
    for _ in range(nt):
        efwd()
    t1e.record(stream)
    for _ in range(nt):
        ebwd()
    t2e.record(stream)
    torch.cuda.synchronize()
    ep_fwd_us = t0e.elapsed_time(t1e) * 1e3 / nt
    ep_bwd_us = t1e.elapsed_time(t2e) * 1e3 / nt
    n_ep = eB * eL * eH * edh
    log(f"mixer epilogue: fwd {ep_fwd_us:.1f} us, bwd {ep_bwd_us:.1f} us")
    del et

    # ---------------- mixer block forward (projections, mixing, epilogue) ----------------
    blk = []
    for Lb in (2048, 8192, 32768):
        pb_ = W.block_inputs(13, 4, Lb, 256, 8, 4, 8, 8, "bf16")
        bt = {k: torch.from_numpy(pb_[k].view(np.int16)).view(torch.bfloat16).to(dev) for k in ("x", "Wu", "Wg", "Wo")}
        bp = [torch.from_numpy(pb_[k]).to(dev) for k in ("gamma", "omega", "amp", "phase", "Ct", "w", "s")]
        del pb_

        dense = tuple(ops.resonator_block_diag_weight(bt[k]) for k in ("Wu", "Wg", "Wo"))

        def block():  # grouped projections (the MFMA projection kernel), drive and gate in one call
            return ops.resonator_block_fwd(bt["x"], bt["Wu"], bt["Wg"], bt["Wo"], *bp[:4], bp[4], 0.5, bp[5], bp[6], 8)

        for _ in range(3):
            block()
        torch.cuda.synchronize()
        reps = 10
        t0e.record(stream)
        for _ in range(reps):
            block()
        t1e.record(stream)
        torch.cuda.synchronize()
        b_us = t0e.elapsed_time(t1e) * 1e3 / reps
        # the same forward replayed from a captured graph (no host issue time)
        bgraph = ops.BlockForwardGraph(bt["x"], bt["Wu"], bt["Wg"], bt["Wo"], *bp[:4], bp[4], 0.5, bp[5], bp[6], 8)
        bgraph.replay()
        torch.cuda.synchronize()
        t0e.record(stream)
        for _ in range(reps):
            bgraph.replay()
        t1e.record(stream)
        torch.cuda.synchronize()
        bg_us = t0e.elapsed_time(t1e) * 1e3 / reps
        del bgraph
        # backward (recomputes the forward's intermediates, then the chain rule)
        dob = torch.randn_like(bt["x"], dtype=torch.float32).to(torch.bfloat16)

        def block_bwd():
            return ops.resonator_block_bwd(bt["x"], bt["Wu"], bt["Wg"], bt["Wo"], *bp[:4], bp[4], 0.5, bp[5], bp[6],
                                           8, dob, dense=dense)

        block_bwd()
        torch.cuda.synchronize()
        t0e.record(stream)
        for _ in range(reps):
            block_bwd()
        t1e.record(stream)
        torch.cuda.synchronize()
        bb_us = t0e.elapsed_time(t1e) * 1e3 / reps

        # a training step that keeps the forward's intermediates: the forward
        # also writes z, the backward skips the recomputation
        def block_step_saved():
            _, sv = ops.resonator_block_fwd(bt["x"], bt["Wu"], bt["Wg"], bt["Wo"], *bp[:4], bp[4], 0.5, bp[5], bp[6], 8,
                                            save=True)
            return ops.resonator_block_bwd(bt["x"], bt["Wu"], bt["Wg"], bt["Wo"], *bp[:4], bp[4], 0.5, bp[5], bp[6],
                                           8, dob, dense=dense, saved=sv)

        block_step_saved()
        torch.cuda.synchronize()
        t0e.record(stream)
        for _ in range(reps):
            block_step_saved()
        t1e.record(stream)
        torch.cuda.synchronize()
        bs_us = t0e.elapsed_time(t1e) * 1e3 / reps
        blk.append({"L": Lb, "fwd_us": b_us, "fwd_graph_us": bg_us, "bwd_us": bb_us, "step_us": b_us + bb_us,
                    "step_saved_us": bs_us,
                    "fwd_tokens_per_s": 4 * Lb / (b_us * 1e-6), "fwd_graph_tokens_per_s": 4 * Lb / (bg_us * 1e-6)})
        log(f"mixer block B4 L={Lb} d256: forward {b_us:.1f} us ({4 * Lb / (b_us * 1e-6) / 1e6:.1f} M tokens/s), "
            f"graph replay {bg_us:.1f} us, backward {bb_us:.1f} us, step with saved intermediates {bs_us:.1f} us")
        del bt, dob

    # ---------------- kernel tail: mixing vs a quadratic causal reference ----------------
    kt = []
    for Lk in (8192, 32768):
        pk = W.random_problem(12, 1, Lk, 256, 8, act="f32", gamma_range=(1e-4, 1.0), gamma_log=True)
        xk = torch.from_numpy(pk["x"]).to(dev)
        prk = [torch.from_numpy(pk[k]).to(dev) for k in ("gamma", "omega", "amp", "phase")]
        ops.resonator_mix_fwd(xk, *prk)
        ops.resonator_quadratic_reference(xk, *prk)
        ops.resonator_fft_reference(xk, *prk)
        torch.cuda.synchronize()
        reps = 20
        t0e.record(stream)
        for _ in range(reps):
            ops.resonator_mix_fwd(xk, *prk)
        t1e.record(stream)
        for _ in range(3):
            ops.resonator_quadratic_reference(xk, *prk)
        t2e.record(stream)
        for _ in range(reps):
            ops.resonator_fft_reference(xk, *prk)
        t3e.record(stream)
        torch.cuda.synchronize()
        mix_us = t0e.elapsed_time(t1e) * 1e3 / reps
        quad_us = t1e.elapsed_time(t2e) * 1e3 / 3
        fft_us = t2e.elapsed_time(t3e) * 1e3 / reps
        kt.append({"L": Lk, "mix_us": mix_us, "quadratic_us": quad_us, "speedup": quad_us / mix_us,
                   "quadratic_TFLOPs": Lk * (Lk + 1) / 2 * 256 * 2 / (quad_us * 1e-6) / 1e12,
                   "fft_us": fft_us, "fft_over_mix": fft_us / mix_us})
        log(f"kernel tail L={Lk}: mixing {mix_us:.1f} us, quadratic reference {quad_us:.0f} us "
            f"(speedup {quad_us / mix_us:.0f}x), FFT convolution {fft_us:.1f} us ({fft_us / mix_us:.1f}x)")
        del xk

    traffic = counter_traffic(n_tok)
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens*ch/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": cfg.name, "B": B, "L": L, "D": D, "M": M,
                   "activations": "bf16 in/out, fp32 accumulate, split-bf16 MFMA operands",
                   "terminal_state": True, "buffer_sets": NSET},
        "fp32_configs": {"workload": "configs 1 and 2, float32 in/out: the step (all kernels of a forward call) and "
                                     "the dominant kernel alone (8 algorithmic bytes per token-channel)",
                         "points": fcfg},
        "copy_GBs": copy_gbs,
        "prefill_sweep": {"workload": "B4 D256 M8 bf16, L = 1K .. 32K (forward kernel GB/s: 4 algorithmic bytes per "
                                      "token-channel); one buffer set per length, so inputs stay in the 256 MB "
                                      "Infinity Cache between calls (the headline line rotates three sets)",
                          "points": sweep},
        "mixer_block": {"workload": "B4 d_model 256, bf16: grouped in-projection (8 groups) to drive and gate in one "
                                    "MFMA projection call, mixing (M8), epilogue (H8 x dh32, K4), grouped out-projection "
                                    "(MFMA); forward, and backward (recomputed forward, then the chain rule with the data "
                                    "gradients from the MFMA data-gradient kernel, the input's three in one pass, and "
                                    "the MFMA weight-gradient kernel); step_us = forward + backward with the "
                                    "recomputation, step_saved_us = forward keeping u, g, y, z + backward on them",
                        "points": blk},
        "kernel_tail": {"workload": "B1 D256 M8 fp32, mixing step (forward kernel) vs the O(L^2) direct "
                                    "causal reference (taps + Toeplitz sum), paper Table 5 protocol, and vs the "
                                    "zero-padded FFT convolution (rocFFT, the paper's prefill form)",
                        "points": kt},
        "decode_multi_step": {"workload": f"{c4.name}: drives known in advance",
                              "k8_us_per_launch": k8_us, "k8_us_per_step": k8_us / 8,
                              "long_steps_per_launch": int(xdec.shape[0]), "long_us_per_step": long_us},
        "decode": {"workload": c4.name, "steps": nsteps,
                   "steps_per_s_eager": 1e6 / dec_eager_us, "us_per_step_eager": dec_eager_us,
                   "steps_per_s_graph": 1e6 / dec_graph_us, "us_per_step_graph": dec_graph_us,
                   "graph_launch_floor_us": floor_us, "graph_over_floor": dec_graph_us / floor_us,
                   "alg_GBs_graph": dec_bytes / (dec_graph_us * 1e-6) / 1e9},
        "train_layer": {"workload": "B8 L8192 D256 M8 bf16 (one of the 6 layers)",
                        "fwd_us": tr_fwd_us, "bwd_us": tr_bwd_us,
                        "bwd_alg_GBs": 8 * 8192 * 256 * 6 / (tr_bwd_us * 1e-6) / 1e9},
        "mixer_epilogue": {"workload": f"B{eB} L{eL} H{eH} dh{edh} K{eK} bf16 (coupling, gate, local path)",
                           "fwd_us": ep_fwd_us, "bwd_us": ep_bwd_us,
                           "fwd_alg_GBs": n_ep * 8 / (ep_fwd_us * 1e-6) / 1e9,
                           "bwd_alg_GBs": n_ep * 14 / (ep_bwd_us * 1e-6) / 1e9},
        "roofline": {"bound": "hbm", "kernel": "fwd_stream_kernel",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "frac_of_copy": achieved / copy_gbs,
                     "traffic": traffic,
                     "alg_bytes_per_launch": alg_bytes, "avg_launch_us": k_avg_ms * 1e3,
                     "ms_per_step_with_kernel_events": ms_step_ev},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
