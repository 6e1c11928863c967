"""Benchmark of the DF-SSM scaffold + int8 LoRA linear on one MI355X.

Headline workload (one "step"): the Mamba-2-1.3B decode sweep at one token --
48 layers x (in_proj 2048->8512, out_proj 4096->2048), rank-64 int8 LoRA,
every output re-quantised as the next input (dfssm_scaffold_lora_chain).
Metric: effective packed-weight GB/s (sign words + LoRA factors + row scales
read per step / step time) and us per layer; the 2048-token prefill in_proj
is measured beside it in int8 TOPS.

Weights are synthetic and seeded (no trained weights exist here).  The sweep
reads 210 MB per step, which fits the 256 MB Infinity Cache, so steps rotate
over several distinct weight copies to keep the measurement cold.

Prints one JSON line.
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

PEAK_HBM_GBS = 8000.0        # MI355X HBM3E
PEAK_I8_TOPS = 5000.0        # MI355X dense int8 MFMA


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--copies", type=int, default=3, help="distinct weight copies rotated per step")
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--no-prefill", action="store_true")
    p.add_argument("--cpu-sample-linears", type=int, default=16)
    return p.parse_args()


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

    # ---- the decode sweep: copies of 96 seeded weight sets -----------------
    shapes = S.sweep_shapes(48)
    copies, arrays, host0 = [], [], None
    for c in range(args.copies):
        hs = S.sweep_weights(48, r=64, variant=c)
        if c == 0:
            host0 = hs
        dl = [{k: dev(v) for k, v in ly.items()} for ly in hs]
        copies.append(dl)
        arrays.append(D.make_layers(dl))
        if c:
            del hs
    weight_bytes = sum(S.weight_bytes(ly) for ly in host0)
    x = S.sweep_input(1)
    q0, s0 = D.quantize_act(dev(x))
    M = 1
    ws_bytes = D.chain_workspace_bytes(arrays[0], M)
    workspace = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    y_all = torch.empty(sum(N for _, N in shapes), dtype=torch.float32, device="cuda")

    def step(i):
        c = i % len(copies)
        D.scaffold_lora_chain(copies[c], q0, s0, y_all=y_all, workspace=workspace, layer_arr=arrays[c])

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(args.steps):
        step(i)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    gbs = weight_bytes / (ms * 1e-3) / 1e9

    # warm (one copy, cache resident) for context
    e0.record()
    for i in range(args.steps):
        step(0)
    e1.record()
    torch.cuda.synchronize()
    ms_warm = e0.elapsed_time(e1) / args.steps

    # ---- prefill: 2048-token in_proj -----------------------------------------
    prefill = None
    if not args.no_prefill:
        pw = {k: dev(v) for k, v in S.config_weights(4).items()}
        xq, xs = D.quantize_act(dev(S.config_activations(4, 2048)))
        yp = torch.empty((2048, 8512), dtype=torch.float32, device="cuda")
        wsp = torch.empty(D.linear_workspace_bytes(2048, 2048, 8512, 64), dtype=torch.uint8, device="cuda")

        def pstep():
            D.scaffold_lora_linear(xq, xs, pw["w_bits"], pw["alpha"], pw["A"], pw["B"], pw["beta"], y=yp,
                                   workspace=wsp)
        for _ in range(3):
            pstep()
        torch.cuda.synchronize()
        e0.record()
        n = 20
        for _ in range(n):
            pstep()
        e1.record()
        torch.cuda.synchronize()
        pms = e0.elapsed_time(e1) / n
        ops = 2.0 * 2048 * 2048 * 8512
        lora_ops = 2.0 * 2048 * 64 * (2048 + 8512)
        prefill = {"workload": "1.3B in_proj prefill M=2048 K=2048 N=8512 r=64", "us": round(pms * 1e3, 2),
                   "scaffold_tops": round(ops / (pms * 1e-3) / 1e12, 1),
                   "algorithmic_tops": round((ops + lora_ops) / (pms * 1e-3) / 1e12, 1),
                   "frac_i8_peak": round(ops / (pms * 1e-3) / 1e12 / PEAK_I8_TOPS, 4)}

    # ---- CPU oracle baseline on a bounded sample ----------------------------
    cpu = None
    if not args.no_cpu:
        import oracle
        if not os.path.exists(oracle.LIB):
            oracle.build()
        o = oracle.get()
        nl = max(2, min(args.cpu_sample_linears, len(host0)))
        q0h, s0h = o.quantize_act(x)
        t = time.perf_counter()
        o.chain(host0[:nl], q0h, s0h)
        dt = time.perf_counter() - t
        sample_bytes = sum(S.weight_bytes(ly) for ly in host0[:nl])
        cpu = {"value": round(sample_bytes / dt / 1e9, 4), "unit": "GB/s", "cores": o.threads(),
               "kind": "oracle",
               "sample": f"first {nl} of the 96 chained linears (M=1), {sample_bytes} weight bytes, {dt:.2f} s"}

    roof_achieved = gbs
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
        "roofline": {"bound": "hbm", "achieved": round(roof_achieved, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(roof_achieved / PEAK_HBM_GBS, 4), "traffic": None},
        "prefill": prefill,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
