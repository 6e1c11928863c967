"""Benchmark of the DF-SSM scaffold + int8 LoRA linear on one MI355X.

Headline workload (one "step"): the Mamba-2-1.3B decode sweep at one token --
48 layers x (in_proj 2048->8512, out_proj 4096->2048), rank-64 int8 LoRA,
every output re-quantised as the next input.  One step is one
dfssm_chain_run, i.e. one launch of the persistent chain kernel, on a
workspace prepared once per weight set (dfssm_chain_prepare, untimed).
Metric: effective packed-weight GB/s (sign words + LoRA factors + row scales
read per step / step time) and us per layer; the 2048-token prefill in_proj
is measured beside it in int8 TOPS, the decode-size single linears in us per
call, the LM head over the 1.3B tied int8 table (103 MB) in GB/s, and the
whole 1.3B decode step (48 layers + LM head, as replayed hipGraphs) in
tokens/s at batch 1, 8, 32, 128 and 512.

Weights are synthetic and seeded (no trained weights exist here).  The sweep
reads 210 MB per step, which fits the 256 MB Infinity Cache, so steps rotate
over several distinct weight copies (630 MB for 3) to keep the measurement
cold.

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0        # MI355X HBM3E
PEAK_I8_TOPS = 5000.0        # MI355X dense int8 MFMA
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "chain_persistent_1p3b_sweep_traffic.txt")
CHAIN_SOURCES = ["paper_2606_10932_amd/csrc/dfssm_chain.hip", "paper_2606_10932_amd/csrc/dfssm_internal.hpp",
                 "paper_2606_10932_amd/csrc/dfssm_persist.hpp"]


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--copies", type=int, default=3, help="distinct weight copies rotated per step")
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--no-prefill", action="store_true")
    p.add_argument("--no-decode", action="store_true", help="skip the single-linear decode-size figures")
    p.add_argument("--no-lm-head", action="store_true", help="skip the LM head figures")
    p.add_argument("--no-model", action="store_true", help="skip the whole-model decode step figures")
    p.add_argument("--model-batches", default="1,8,32,128,512", help="batch sizes of the decode step figures")
    p.add_argument("--model-i4-batches", default="1,32",
                   help="batch sizes of the decode step figures with int4 LoRA factors")
    p.add_argument("--no-diag", action="store_true", help="skip the chain's stream and exchange floor diagnostics")
    p.add_argument("--no-i4-sweep", action="store_true", help="skip the decode sweep with int4 LoRA factors")
    p.add_argument("--cpu-seconds", type=float, default=12.0, help="minimum CPU oracle sample time")
    p.add_argument("--cpu-single-seconds", type=float, default=4.0,
                   help="minimum single-thread CPU oracle sample time")
    p.add_argument("--copy-calibration-mib", type=int, default=0,
                   help="run one plain device copy of this size first (for HBM counter scaling)")
    return p.parse_args()


def chain_source_digest() -> str:
    h = hashlib.sha256()
    for rel in CHAIN_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic():
    """(L2-miss bytes, DRAM-request bytes) per chain launch from the committed
    counter summary; (None, None) when it is missing or was taken on other
    kernel sources."""
    try:
        kv = {}
        with open(TRAFFIC_FILE) as f:
            for line in f:
                if ":" in line and not line.startswith("#"):
                    k, v = line.split(":", 1)
                    kv[k.strip()] = v.strip()
        if kv.get("chain_source_sha256") != chain_source_digest():
            return None, None
        return int(float(kv["l2_miss_bytes_per_launch"])), int(float(kv["dram_req_bytes_per_launch"]))
    except (OSError, KeyError, ValueError):
        return None, None


def host_cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (this library has no "
              f"multi-GPU path)", file=sys.stderr)
        sys.exit(2)
    import torch
    import dfssm_synth as S
    import paper_2606_10932_amd as D

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)

    def dev(a):
        a = a.view(np.int32) if a.dtype == np.uint32 else a
        return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")

    if args.copy_calibration_mib:
        n = args.copy_calibration_mib << 20
        a = torch.ones(n // 4, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    # ---- the decode sweep: copies of 96 seeded weight sets -----------------
    shapes = S.sweep_shapes(48)
    M = 1
    copies, arrays, workspaces, host0 = [], [], [], None
    for c in range(args.copies):
        hs = S.sweep_weights(48, r=64, variant=c)
        if c == 0:
            host0 = hs
        dl = [{k: dev(v) for k, v in ly.items()} for ly in hs]
        arr = D.make_layers(dl)
        ws = torch.zeros(D.chain_workspace_bytes(arr, M), dtype=torch.uint8, device="cuda")
        D.chain_prepare(arr, M, ws)
        copies.append(dl)
        arrays.append(arr)
        workspaces.append(ws)
        if c:
            del hs
    weight_bytes = sum(S.weight_bytes(ly) for ly in host0)
    x = S.sweep_input(1)
    q0, s0 = D.quantize_act(dev(x))
    y_all = torch.empty(sum(N for _, N in shapes), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()

    def step(i):
        c = i % len(copies)
        D.chain_run(arrays[c], q0, s0, y_all, workspaces[c], stream=stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    # timed region: K launches back to back; an event pair around each launch
    # (on the launch stream) gives the kernel's own duration
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for i in range(args.steps):
        ev[i][0].record(stream)
        step(i)
        ev[i][1].record(stream)
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / args.steps
    launch_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    status = max(D.chain_status(arrays[c], M, workspaces[c]) for c in range(len(copies)))
    if status:
        print(f"chain status word {status:#x}: a bounded wait gave up", file=sys.stderr)
        sys.exit(3)
    gbs = weight_bytes / (ms * 1e-3) / 1e9
    launch_gbs = weight_bytes / (launch_ms * 1e-3) / 1e9

    # warm (one copy, cache resident) for context
    t0.record(stream)
    for i in range(args.steps):
        step(0)
    t1.record(stream)
    torch.cuda.synchronize()
    ms_warm = t0.elapsed_time(t1) / args.steps

    # ---- diagnostics: the two floors under the chain ---------------------------
    diag = None
    if not args.no_diag:
        # (1) the same layers' operand loads alone, through the chain's own
        #     loading schedule (no arithmetic, no exchange): the stream floor
        def sstep(i):
            c = i % len(copies)
            D.chain_stream_floor(arrays[c], workspaces[c], stream=stream)
        for i in range(3):
            sstep(i)
        sev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        torch.cuda.synchronize()
        for i in range(args.steps):
            sev[i][0].record(stream)
            sstep(i)
            sev[i][1].record(stream)
        torch.cuda.synchronize()
        stream_ms = float(np.median([a.elapsed_time(b) for a, b in sev]))
        if max(D.chain_status(arrays[c], M, workspaces[c]) for c in range(len(copies))):
            print("chain stream diagnostic: status word set", file=sys.stderr)
            sys.exit(3)
        stream_gbs = weight_bytes / (stream_ms * 1e-3) / 1e9
        # (2) the chain on 96 tiny linears (K = N = 256, r = 4, 12 KB of
        #     weights each): what is left is the per-linear exchange and
        #     compute latency
        tiny = [S.weights(256, 256, 4, key=(60, i)) for i in range(96)]
        tiny_bytes = sum(S.weight_bytes(ly) for ly in tiny)
        tarr = D.make_layers([{k: dev(v) for k, v in ly.items()} for ly in tiny])
        tws = torch.zeros(D.chain_workspace_bytes(tarr, 1), dtype=torch.uint8, device="cuda")
        D.chain_prepare(tarr, 1, tws)
        tq, ts = D.quantize_act(dev(S.activations(1, 256, key=(61,))))
        ty = torch.empty(96 * 256, dtype=torch.float32, device="cuda")
        for i in range(3):
            D.chain_run(tarr, tq, ts, ty, tws, stream=stream)
        tev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        torch.cuda.synchronize()
        for i in range(args.steps):
            tev[i][0].record(stream)
            D.chain_run(tarr, tq, ts, ty, tws, stream=stream)
            tev[i][1].record(stream)
        torch.cuda.synchronize()
        tiny_ms = float(np.median([a.elapsed_time(b) for a, b in tev]))
        if D.chain_status(tarr, 1, tws):
            print("tiny chain diagnostic: status word set", file=sys.stderr)
            sys.exit(3)
        diag = {
            "stream_floor": {
                "workload": "the sweep's 96 linears, operand loads only (chain_stream: the persistent chain's "
                            "direct-to-LDS schedule, no arithmetic, no exchange), 3 weight copies rotated",
                "us_per_sweep": round(stream_ms * 1e3, 2), "gbs": round(stream_gbs, 1),
                "frac_hbm_peak": round(stream_gbs / PEAK_HBM_GBS, 4),
                "chain_over_floor": round(launch_ms / stream_ms, 2)},
            "exchange_floor": {
                "workload": "persistent chain of 96 linears K=N=256, r=4, M=1 (%d B of weights in all)" % tiny_bytes,
                "us_per_sweep": round(tiny_ms * 1e3, 2), "us_per_linear": round(tiny_ms * 1e3 / 96, 3)},
            "hop": {
                "workload": "one agent-scope word passed between two workgroups on two XCDs "
                            "(dfssm_exchange_pingpong), median over the pairs",
                "round_trip_ns_1_pair": round(D.exchange_pingpong(1, 2000), 1),
                "round_trip_ns_128_pairs": round(D.exchange_pingpong(128, 2000), 1),
                "round_trip_ns_release_acquire": round(D.exchange_pingpong(1, 200, fence=True), 1)},
        }
        del tarr, tws, ty

    # ---- the same sweep with int4 LoRA factors (Table 4): 3 rotating copies,
    #      the same persistent kernel reading the packed factors --------------
    sweep_i4 = None
    if not args.no_i4_sweep:
        arrs4, wss4, keep4, bytes4 = [], [], [], 0
        for c in range(args.copies):
            hs4 = [S.weights_i4(K, N, 64, key=(70, i, c)) for i, (K, N) in enumerate(shapes)]
            if c == 0:
                bytes4 = sum(int(sum(ly[k].nbytes for k in ("w_bits", "alpha", "A4", "B4", "beta"))) for ly in hs4)
            dl4 = [{k: dev(v) for k, v in ly.items()} for ly in hs4]
            a4 = D.make_layers(dl4)
            w4 = torch.zeros(D.chain_workspace_bytes(a4, M), dtype=torch.uint8, device="cuda")
            D.chain_prepare(a4, M, w4)
            arrs4.append(a4)
            wss4.append(w4)
            keep4.append(dl4)
            del hs4
        for i in range(max(args.warmup, 2)):
            D.chain_run(arrs4[i % len(arrs4)], q0, s0, y_all, wss4[i % len(arrs4)], stream=stream)
        ev4 = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        torch.cuda.synchronize()
        t0.record(stream)
        for i in range(args.steps):
            ev4[i][0].record(stream)
            D.chain_run(arrs4[i % len(arrs4)], q0, s0, y_all, wss4[i % len(arrs4)], stream=stream)
            ev4[i][1].record(stream)
        t1.record(stream)
        torch.cuda.synchronize()
        ms4 = t0.elapsed_time(t1) / args.steps
        launch4 = float(np.mean([a.elapsed_time(b) for a, b in ev4]))
        if max(D.chain_status(arrs4[c], M, wss4[c]) for c in range(len(arrs4))):
            print("int4 chain status word set: a bounded wait gave up", file=sys.stderr)
            sys.exit(3)
        sweep_i4 = {"workload": "Mamba-2-1.3B decode sweep, M=1, 96 linears, int4 LoRA factors r=64, "
                                f"{len(arrs4)} weight copies rotated",
                    "ms_per_step": round(ms4, 4), "avg_launch_us": round(launch4 * 1e3, 2),
                    "weight_bytes": bytes4, "gbs": round(bytes4 / (ms4 * 1e-3) / 1e9, 1),
                    "frac_hbm_peak": round(bytes4 / (ms4 * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
                    "int8_sweep_ms_per_step": round(ms, 4)}
        del arrs4, wss4, keep4

    # ---- prefill: 2048-token in_proj -----------------------------------------
    prefill = None
    if not args.no_prefill:
        pw = {k: dev(v) for k, v in S.config_weights(4).items()}
        xq, xs = D.quantize_act(dev(S.config_activations(4, 2048)))
        yp = torch.empty((2048, 8512), dtype=torch.float32, device="cuda")
        wsp = D.linear_workspace(2048, 2048, 8512, 64)

        def pstep():
            D.scaffold_lora_linear(xq, xs, pw["w_bits"], pw["alpha"], pw["A"], pw["B"], pw["beta"], y=yp,
                                   workspace=wsp, stream=stream)
        for _ in range(3):
            pstep()
        torch.cuda.synchronize()
        t0.record(stream)
        n = 20
        for _ in range(n):
            pstep()
        t1.record(stream)
        torch.cuda.synchronize()
        pms = t0.elapsed_time(t1) / n
        ops = 2.0 * 2048 * 2048 * 8512
        lora_ops = 2.0 * 2048 * 64 * (2048 + 8512)
        prefill = {"workload": "1.3B in_proj prefill M=2048 K=2048 N=8512 r=64 (down-projection + scaffold "
                               "launches)", "us": round(pms * 1e3, 2),
                   "scaffold_tops": round(ops / (pms * 1e-3) / 1e12, 1),
                   "algorithmic_tops": round((ops + lora_ops) / (pms * 1e-3) / 1e12, 1),
                   "frac_i8_peak": round(ops / (pms * 1e-3) / 1e12 / PEAK_I8_TOPS, 4)}

    # ---- single linears at decode sizes ---------------------------------------
    # Per call: q, s -> y on the automatic path (the one-launch few-token
    # MFMA kernel at these sizes).  The calls of one graph replay walk
    # over distinct copies of the weights, about 600 MB in all, so every call
    # meets its weights outside the 256 MB Infinity Cache; the graph removes
    # the host's launch cost from the measurement.
    def read_floors(nbytes, ncall):
        """The floor under a single linear of nbytes of weights: one launch
        reading nbytes (dfssm_read_floor), over ncall distinct buffers so
        every read is cold, replayed from a graph as the linears are; and
        the same graph of empty launches."""
        nb16 = (nbytes + 15) // 16 * 16
        bufs = [torch.empty(nb16, dtype=torch.uint8, device="cuda") for _ in range(ncall)]
        sink = torch.zeros(D.read_floor_sink_words(nb16), dtype=torch.int32, device="cuda")
        out = {}
        for label, nb in (("floor_us_read", nb16), ("floor_us_launch", 0)):
            def calls():
                for b in bufs:
                    D.read_floor(b, sink, nbytes=nb)
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                calls()
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=side):
                    calls()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            reps = 3
            t0.record(stream)
            for _ in range(reps):
                g.replay()
            t1.record(stream)
            torch.cuda.synchronize()
            out[label] = round(t0.elapsed_time(t1) * 1e3 / (reps * ncall), 2)
            del g
        del bufs
        return out

    decode = None
    if not args.no_decode:
        decode = []
        for cfg, name, Ms in ((0, "Mamba-2-130M in_proj K=768 N=3352 r=16", (1,)),
                              (1, "Mamba-2-1.3B in_proj K=2048 N=8512 r=64", (1,)),
                              (2, "Mamba-2-1.3B out_proj K=4096 N=2048 r=64", (1, 4, 8, 16, 32))):
            hw = S.config_weights(cfg)
            wb = S.weight_bytes(hw)
            base = {k: dev(v) for k, v in hw.items()}
            ncall = int(np.ceil(600e6 / wb))
            cps = [base] + [{k: v.clone() for k, v in base.items()} for _ in range(ncall - 1)]
            K, N = hw["A"].shape[1], hw["w_bits"].shape[0]
            r = hw["A"].shape[0]
            for m in Ms:
                qd, sd = D.quantize_act(dev(S.config_activations(cfg, m)))
                yd = torch.empty((m, N), dtype=torch.float32, device="cuda")
                wsd = D.linear_workspace(m, K, N, r)

                def calls():
                    for c in cps:
                        D.scaffold_lora_linear(qd, sd, c["w_bits"], c["alpha"], c["A"], c["B"], c["beta"], y=yd,
                                               workspace=wsd)
                side = torch.cuda.Stream()
                side.wait_stream(torch.cuda.current_stream())
                with torch.cuda.stream(side):
                    calls()
                    g = torch.cuda.CUDAGraph()
                    with torch.cuda.graph(g, stream=side):
                        calls()
                torch.cuda.synchronize()
                g.replay()
                torch.cuda.synchronize()
                reps = 3
                t0.record(stream)
                for _ in range(reps):
                    g.replay()
                t1.record(stream)
                torch.cuda.synchronize()
                us = t0.elapsed_time(t1) * 1e3 / (reps * ncall)
                del g
                # warm: the same number of calls, all on the first copy (its
                # weights stay in the Infinity Cache and L2)

                def calls_warm():
                    for _ in cps:
                        D.scaffold_lora_linear(qd, sd, base["w_bits"], base["alpha"], base["A"], base["B"],
                                               base["beta"], y=yd, workspace=wsd)
                with torch.cuda.stream(side):
                    calls_warm()
                    g = torch.cuda.CUDAGraph()
                    with torch.cuda.graph(g, stream=side):
                        calls_warm()
                torch.cuda.synchronize()
                g.replay()
                torch.cuda.synchronize()
                t0.record(stream)
                for _ in range(reps):
                    g.replay()
                t1.record(stream)
                torch.cuda.synchronize()
                us_warm = t0.elapsed_time(t1) * 1e3 / (reps * ncall)
                fig = {"workload": f"{name} M={m}", "us_per_call": round(us, 2),
                       "us_per_call_warm": round(us_warm, 2),
                       "weight_gbs": round(wb / (us * 1e-6) / 1e9, 1), "weight_bytes": wb,
                       "path": "few-token MFMA (one launch)", "lora": "int8"}
                if m == 1 and cfg > 0:
                    # the floor: a cold one-launch read of the same bytes
                    fig.update(read_floors(wb, ncall))
                decode.append(fig)
                del g
            del cps, base
        # the same projections with int4 LoRA factors (packed bytes read by
        # the few-token kernel), same method
        for cfg, name, Ms in ((1, "Mamba-2-1.3B in_proj K=2048 N=8512 r=64", (1,)),
                              (2, "Mamba-2-1.3B out_proj K=4096 N=2048 r=64", (1, 32))):
            c = S.CONFIGS[cfg]
            hw = S.weights_i4(c.K, c.N, c.r, key=(cfg, 0, 0, 4))
            wb = int(sum(hw[k].nbytes for k in ("w_bits", "alpha", "A4", "B4", "beta")))
            base = {k: dev(v) for k, v in hw.items()}
            ncall = int(np.ceil(600e6 / wb))
            cps = [base] + [{k: v.clone() for k, v in base.items()} for _ in range(ncall - 1)]
            for m in Ms:
                qd, sd = D.quantize_act(dev(S.config_activations(cfg, m)))
                yd = torch.empty((m, c.N), dtype=torch.float32, device="cuda")
                # a workspace holds zeros before its first use (its epoch words)
                wsd = torch.zeros(int(D.lib.dfssm_linear_i4_workspace_bytes(m, c.K, c.N, c.r)), dtype=torch.uint8,
                                  device="cuda")

                def calls4():
                    for cc in cps:
                        D.scaffold_lora_linear_i4(qd, sd, cc["w_bits"], cc["alpha"], cc["A4"], cc["B4"], cc["beta"],
                                                  y=yd, workspace=wsd)
                side = torch.cuda.Stream()
                side.wait_stream(torch.cuda.current_stream())
                with torch.cuda.stream(side):
                    calls4()
                    g = torch.cuda.CUDAGraph()
                    with torch.cuda.graph(g, stream=side):
                        calls4()
                torch.cuda.synchronize()
                g.replay()
                torch.cuda.synchronize()
                reps = 3
                t0.record(stream)
                for _ in range(reps):
                    g.replay()
                t1.record(stream)
                torch.cuda.synchronize()
                us = t0.elapsed_time(t1) * 1e3 / (reps * ncall)
                decode.append({"workload": f"{name} M={m}", "us_per_call": round(us, 2),
                               "weight_gbs": round(wb / (us * 1e-6) / 1e9, 1), "weight_bytes": wb,
                               "path": "few-token MFMA (one launch)", "lora": "int4"})
                del g
            del cps, base

    # ---- LM head on the tied int8 embedding ---------------------------------
    # logits of M tokens over the 1.3B vocabulary (50,280 x 2048 int8 table,
    # 103 MB).  One graph replay walks over 4 distinct copies of the table
    # (412 MB), so every call streams its table from HBM.
    lm, table0 = None, None
    if not args.no_lm_head:
        lm = []
        Eh, sch = S.embedding(S.VOCAB_1P3B, S.D_MODEL_1P3B, key=(40,))
        tb = Eh.nbytes + sch.nbytes
        tabs = [(dev(Eh), dev(sch))]
        tabs += [(tabs[0][0].clone(), tabs[0][1].clone()) for _ in range(3)]
        del Eh
        for m in (1, 4, 64, 512):
            qd, sd = D.quantize_act(dev(S.activations(m, S.D_MODEL_1P3B, key=(45,))))
            lg = torch.empty((m, S.VOCAB_1P3B), dtype=torch.float32, device="cuda")

            def lcalls():
                for E_, sc_ in tabs:
                    D.lm_head(qd, sd, E_, sc_, logits=lg)
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                lcalls()
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=side):
                    lcalls()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            reps = 5
            t0.record(stream)
            for _ in range(reps):
                g.replay()
            t1.record(stream)
            torch.cuda.synchronize()
            us = t0.elapsed_time(t1) * 1e3 / (reps * len(tabs))
            lm.append({"workload": f"LM head 50280 x 2048 int8 table, M={m}", "us_per_call": round(us, 2),
                       "table_gbs": round(tb / (us * 1e-6) / 1e9, 1),
                       "frac_hbm_peak": round(tb / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4), "table_bytes": tb,
                       "int8_tops": round(2.0 * m * S.VOCAB_1P3B * S.D_MODEL_1P3B / (us * 1e-6) / 1e12, 1),
                       "kernel": "GEMV passes" if m < 8 else "matrix cores"})
            del g
        table0 = tabs[0]
        del tabs

    # ---- the whole decode step of the 1.3B model ----------------------------
    # dfssm_mamba2_decode_step (gather, 48 x [norm, in_proj, conv + SSM step,
    # gated norm, out_proj], final norm, LM head) captured as four graphs,
    # one per ring slot, replayed token after token on zero-initialised state.
    # The linears are weight copy 0 of the sweep, the table the LM head's.
    model_fig = None
    if not args.no_model:
        if table0 is None:
            Eh, sch = S.embedding(S.VOCAB_1P3B, S.D_MODEL_1P3B, key=(40,))
            table0 = (dev(Eh), dev(sch))
            del Eh
        layers = []
        for l in range(48):
            lp = {k: dev(v) for k, v in S.mamba_params(2048, key=(150, l)).items()}
            lp["in_proj"], lp["out_proj"] = copies[0][2 * l], copies[0][2 * l + 1]
            layers.append(lp)
        norm_f = dev(np.random.default_rng(151).uniform(0.8, 1.2, 2048).astype(np.float32))
        mdl = D.Mamba2(table0[0], table0[1], norm_f, layers)
        param_bytes = 2048 * 4 + sum(v.numel() * 4 for lp in layers for k, v in lp.items()
                                     if k not in ("in_proj", "out_proj"))
        table_bytes = table0[0].numel() + table0[1].numel() * 4
        model_fig = []

        def time_model(mdl, Mb, wbytes, label, prepare=True):
            ring, state = mdl.new_state(Mb)
            ws_m = mdl.workspace(Mb, prepare=prepare)
            tok = dev(S.tokens(Mb, S.VOCAB_1P3B, key=(152, Mb)))
            lg = torch.empty((Mb, S.VOCAB_1P3B), dtype=torch.float32, device="cuda")
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            graphs = []
            with torch.cuda.stream(side):
                mdl.decode_step(tok, 0, ring, state, ws_m, logits=lg)
                for ph in range(4):
                    g = torch.cuda.CUDAGraph()
                    with torch.cuda.graph(g, stream=side):
                        mdl.decode_step(tok, ph, ring, state, ws_m, logits=lg)
                    graphs.append(g)
            torch.cuda.synchronize()
            for tt in range(1, 5):
                graphs[tt % 4].replay()
            torch.cuda.synchronize()
            n = 12
            t0.record(stream)
            for tt in range(5, 5 + n):
                graphs[tt % 4].replay()
            t1.record(stream)
            torch.cuda.synchronize()
            ms_tok = t0.elapsed_time(t1) / n
            # bytes a step must move at least: weights, table, parameters,
            # the SSM state read and written, the ring (3 slots read, 1 written)
            step_bytes = wbytes + table_bytes + param_bytes + 2 * state.numel() * 4 + ring.numel() * 4
            path = "one persistent launch for the 48 layers" if mdl.fused_path(Mb, ws_m) else "per-kernel sequence"
            model_fig.append({"workload": f"Mamba-2-1.3B decode step, batch {Mb}, 48 layers + LM head{label}",
                              "path": path, "ms_per_step": round(ms_tok, 4), "tokens_per_s": round(Mb / (ms_tok * 1e-3), 1),
                              "us_per_layer": round(ms_tok * 1e3 / 48, 2),
                              "bytes_per_step": int(step_bytes),
                              "effective_gbs": round(step_bytes / (ms_tok * 1e-3) / 1e9, 1)})
            del graphs, g, ring, state, ws_m, lg
            torch.cuda.synchronize()

        for Mb in [int(v) for v in args.model_batches.split(",") if v]:
            time_model(mdl, Mb, weight_bytes, "")
            if Mb == 1:
                # the same step on an unprepared workspace: the per-kernel
                # sequence, for comparison
                time_model(mdl, Mb, weight_bytes, "", prepare=False)
        # the same model with int4 LoRA factors (r = 64) in every projection
        i4_batches = [int(v) for v in args.model_i4_batches.split(",") if v]
        if i4_batches:
            del mdl
            layers4, wbytes4 = [], 0
            for l, lp in enumerate(layers):
                lp4 = {k: v for k, v in lp.items() if k not in ("in_proj", "out_proj")}
                for j, (pj, K, N) in enumerate((("in_proj", 2048, 8512), ("out_proj", 4096, 2048))):
                    hw = S.weights_i4(K, N, 64, key=(153, l, j))
                    wbytes4 += sum(v.nbytes for v in hw.values())
                    lp4[pj] = {k: dev(v) for k, v in hw.items()}
                layers4.append(lp4)
            mdl = D.Mamba2(table0[0], table0[1], norm_f, layers4)
            for Mb in i4_batches:
                time_model(mdl, Mb, wbytes4, ", int4 LoRA")
            del layers4
        del mdl, layers

    # ---- CPU oracle baseline on a bounded sample ----------------------------
    cpu = None
    if not args.no_cpu:
        import oracle
        if not os.path.exists(oracle.LIB):
            oracle.build()
        o = oracle.get()
        q0h, s0h = o.quantize_act(x)
        reps, t = 0, time.perf_counter()
        while True:
            o.chain(host0, q0h, s0h)
            reps += 1
            dt = time.perf_counter() - t
            if dt >= args.cpu_seconds:
                break
        cpu = {"value": round(reps * weight_bytes / dt / 1e9, 4), "unit": "GB/s", "cores": o.threads(),
               "kind": "oracle",
               "sample": f"the full 96-linear sweep (weight copy 0, same input) run {reps} times in {dt:.1f} s",
               "us_per_layer": round(dt / reps / 48 * 1e6, 1), "host_cpu": host_cpu_model(),
               "host_cpus_visible": os.cpu_count()}
        def timed(fn, seconds):
            n, t0h = 0, time.perf_counter()
            while True:
                fn()
                n += 1
                el = time.perf_counter() - t0h
                if el >= seconds:
                    return el / n, n
        # the same oracle on one thread
        threads = o.threads()
        o.set_threads(1)
        reps1, t = 0, time.perf_counter()
        while True:
            o.chain(host0, q0h, s0h)
            reps1 += 1
            dt1 = time.perf_counter() - t
            if dt1 >= args.cpu_single_seconds:
                break
        o.set_threads(threads)
        cpu["single_thread"] = {"value": round(reps1 * weight_bytes / dt1 / 1e9, 4), "unit": "GB/s", "cores": 1,
                                "us_per_layer": round(dt1 / reps1 / 48 * 1e6, 1),
                                "sample": f"the full 96-linear sweep run {reps1} times in {dt1:.1f} s on one thread"}

        # the single linears of the other workloads, on one thread and on all;
        # the 2048-token prefill on a 64-token sample (rows are independent,
        # so its time scales by 2048/64)
        def one_cfg(cfg, m, sample_m, seconds):
            hw = S.config_weights(cfg)
            qc, sc = o.quantize_act(S.config_activations(cfg, sample_m))
            out = {}
            for label, nt in (("us_1_thread", 1), ("us_all_threads", threads)):
                o.set_threads(nt)
                per, n = timed(lambda: o.linear(qc, sc, **hw), seconds)
                out[label] = round(per * 1e6 * m / sample_m, 1)
            o.set_threads(threads)
            return out
        cfgs = []
        for cfg, m, sm in ((0, 1, 1), (1, 1, 1), (2, 1, 1), (2, 4, 4), (2, 8, 8), (2, 16, 16), (2, 32, 32),
                           (4, 2048, 64)):
            e = {"config": f"c{cfg}", "M": m}
            e.update(one_cfg(cfg, m, sm, 0.6))
            if sm != m:
                e["sample"] = f"{sm} of the {m} tokens, time scaled by {m // sm}"
            cfgs.append(e)
        cpu["linears"] = cfgs

        # the oracle beside the other measured kernels: the LM head at one
        # token on the 1.3B table, and one decode layer at batch 1
        Eh, sch = S.embedding(S.VOCAB_1P3B, S.D_MODEL_1P3B, key=(40,))
        qh, sh = o.quantize_act(S.activations(1, S.D_MODEL_1P3B, key=(45,)))
        per, n = timed(lambda: o.lm_head(qh, sh, Eh, sch), 2.0)
        cpu["lm_head_m1_us"] = round(per * 1e6, 1)
        cpu["lm_head_sample"] = f"LM head, M=1, 50,280 x 2048 table, {n} calls"
        del Eh
        lp = S.mamba_params(2048, key=(150, 0))
        st = S.mamba_state(1, 2048, key=(150,))
        u0 = S.residual(1, 2048, key=(150,))
        w_in, w_out = host0[0], host0[1]

        def layer():
            u, _, q1, s1 = o.add_rmsnorm_quant(u0, lp["norm_w"], 1e-5)
            zx = o.linear(q1, s1, **w_in)["y32"]
            y, _, _, _ = o.ssm_step(zx, st["conv_state"], st["ssm_state"], lp["conv_w"], lp["conv_b"],
                                    lp["dt_bias"], lp["A_log"], lp["D"], 4096, 128, 64)
            _, q2, s2 = o.gate_norm_quant(y, zx[:, :4096], lp["gate_w"], 1e-5)
            return o.linear(q2, s2, **w_out)["y32"]
        per, n = timed(layer, 3.0)
        cpu["decode_layer_m1_us"] = round(per * 1e6, 1)
        cpu["decode_layer_sample"] = (f"one 1.3B decode layer at batch 1 (residual norm, in_proj, conv + SSM step, "
                                      f"gated norm, out_proj), {n} runs")

    traffic, dram_bytes = measured_traffic()
    out = {
        "metric": "effective packed-weight GB/s (1.3B decode sweep, M=1)",
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "us_per_layer": round(ms * 1e3 / 48, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i8/u1 (int32/int64 accumulate, fp32 epilogue)",
        "data": "synthetic (seeded Mamba-2-1.3B-shaped weights and activations)",
        "config": {"workload": "Mamba-2-1.3B decode sweep: 48 x (in_proj 2048->8512, out_proj 4096->2048), "
                               "r=64 int8 LoRA, M=1, each output re-quantised",
                   "weight_bytes_per_step": weight_bytes, "weight_copies_rotated": len(copies),
                   "warm_ms_per_step": round(ms_warm, 4)},
        "roofline": {"bound": "hbm", "kernel": "chain_persistent", "achieved": round(launch_gbs, 2),
                     "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(launch_gbs / PEAK_HBM_GBS, 4),
                     "traffic": traffic, "avg_launch_us": round(launch_ms * 1e3, 2),
                     "traffic_is": "L2-miss bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-scaled): the "
                                   "Infinity Cache or HBM serves them",
                     "dram_req_bytes": dram_bytes,
                     "algorithmic_bytes_per_launch": weight_bytes},
        "prefill": prefill,
        "decode_linears": decode,
        "lm_head": lm,
        "decode_step": model_fig,
        "cpu_baseline": cpu,
        "diagnostics": diag,
        "sweep_int4_lora": sweep_i4,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
