#!/usr/bin/env python3
"""Benchmark of one GPU's share of a DSP spatial-temporal block on MI355X.

One step is one pass over the whole hot path, each piece at its own synthetic
workload (video-latent shapes of the 720M model: C=1152, 16 heads of 72):

  switch    dsp_switch of a 1 x 64 x 4096 x 1152 bf16 T-shard into 8 chunks
  switch_inv  the inverse switch: the 1 x 4096 x 64 x 1152 (B,S,T,C) tensor into
            8 chunks along T
  spatial   dsp_spatial_attn,  B=2, T=16,  S=4096 (attention over S)
  temporal  dsp_temporal_attn, B=2, S=512, T=128  (attention over T)
  block     dsp_st_block_forward, B=1, T=32, S=1024, MLP 4608 (LN, QKV,
            spatial attention, out-proj, switch, LN, QKV, temporal attention,
            out-proj, LN, MLP with GELU, residuals)
and, timed separately after the steps (not part of a step):
  exchange  dsp_exchange_unpack among 8 ranks simulated on this GPU, each rank
            holding one such shard's packed switch output (8 x 604 MB in and out)
  temporal_strided  the temporal workload read and written in the unswitched
            (B, T, S, C) layout through dsp_attn_strided
  switch_k3 dsp_switch of the same shard seen as K = 3 sequence dims,
            1 x 64 x 64 x 64 x 1152 (T x H x W), T -> H into 8 chunks
  split     dsp_split of that shard along S into 8, one rank's slice
  gather    dsp_gather of 8 shards 1 x 512 x 64 x 1152 along T (604 MB out)
  attn_bwd_spatial / attn_bwd_temporal  dsp_attn_bwd (dq, dk, dv) of the
            spatial and temporal workloads, given o and the row log-sum-exp
            from dsp_attn_fwd_lse; counted as 10 L^2 D flops per unit (the
            five L x L x D products of the gradient)
  block_train_fwd / block_bwd  dsp_st_block_forward_train (the block keeping
            its activations) and dsp_st_block_backward (dx and every weight
            gradient) on the block workload; the backward counted as twice
            the forward's GEMM flops (dx and dW) plus 10 L^2 D per attention unit

The headline value is the combined attention throughput
(F_spatial + F_temporal) / (t_spatial + t_temporal) in TFLOP/s with
F = 4 L^2 D per (unit) -- useful flops only, no padding, no softmax.  The
switch is reported in GB/s of bytes read + written.  Per-kernel times are HIP
events recorded on the stream the kernels run on, averaged over the timed
steps.  Inputs are resident in HBM before timing starts.

Prints ONE JSON line.  Only one GPU is used; --gpus N with N > 1 exits.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBPS = 8000.0           # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PROBE_ITERS = 5000               # MFMA probe: 8 * 5000 MFMAs per wave, about 7 ms per launch

METRIC = "spatial+temporal attn TFLOP/s (% MFMA peak); dsp_switch GB/s (% HBM peak)"


def attn_flops(units: int, L: int, D: int) -> float:
    return 4.0 * units * L * L * D


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0,
                    help="approximate seconds of oracle work for the CPU baseline")
    ap.add_argument("--traffic", default=os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                                      "profiles", "attention_hbm_traffic.txt"),
                    help="rocprofv3 summary with the measured HBM bytes per launch of the "
                         "spatial kernel; used only while the kernel source is unchanged")
    ap.add_argument("--only", default=None,
                    choices=["switch", "switch_inv", "spatial", "temporal", "block", "exchange",
                             "temporal_strided", "switch_k3", "split", "gather", "copy",
                             "attn_bwd_spatial", "attn_bwd_temporal", "block_train_fwd", "block_bwd",
                             "mfma_probe", "tiny_chain", "tiny_chain_graph"],
                    help="run a single part (for profiling); prints per-kernel times only. "
                         "'copy' is dsp_switch with from_dim == to_dim on the switch tensor: a "
                         "plain 604 MB copy used to calibrate traffic counters")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this build runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(the inter-GPU exchange of the switch is out of scope)", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2403_10266_amd as dsp
    import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()

    def to_dev(a, dt):
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
        return (t.to(torch.bfloat16) if dt == "bf16" else t).to(dev)

    W = synth.WORKLOADS
    ws, wsp, wtp, wbl = (W["switch_bf16_T64_S4096"], W["spatial_bf16_B2_T16_S4096"],
                         W["temporal_bf16_B2_S512_T128"], W["block_bf16_B1_T32_S1024"])
    wanted = {args.only} if args.only else {"switch", "spatial", "temporal", "block", "exchange",
                                            "temporal_strided", "switch_k3", "split", "gather",
                                            "attn_bwd_spatial", "attn_bwd_temporal", "block_train_fwd",
                                            "block_bwd"}
    if wanted & {"block_train_fwd", "block_bwd"}:
        wanted.add("block")
    if "attn_bwd_spatial" in wanted:
        wanted.add("spatial")
    if "attn_bwd_temporal" in wanted:
        wanted.add("temporal")
    if wanted & {"copy", "switch_inv", "exchange", "switch_k3", "split", "gather"}:
        wanted.add("switch")
    if "temporal_strided" in wanted:
        wanted.add("temporal")
    t = {}
    # ---- inputs (seeded, synthetic), resident in HBM before timing
    if "switch" in wanted:
        t["x_sw"] = to_dev(synth.switch_input(ws), "bf16")
        t["y_sw"] = torch.empty((ws.n_chunks, ws.B, ws.S // ws.n_chunks, ws.T, ws.C),
                                dtype=torch.bfloat16, device=dev)
        # the inverse switch (S -> T): the (B, S, T, C) tensor into chunks along T
        t["x_inv"] = t["x_sw"].permute(0, 2, 1, 3).contiguous()
        t["y_inv"] = torch.empty((ws.n_chunks, ws.B, ws.T // ws.n_chunks, ws.S, ws.C),
                                 dtype=torch.bfloat16, device=dev)
    if "exchange" in wanted:
        # N = n_chunks ranks, each holding one switch-shard's packed output
        # (distinct contents; a copy's speed does not depend on the values)
        dsp.dsp_switch(t["x_sw"], 1, 2, ws.n_chunks, out=t["y_sw"])
        t["ex_in"] = [t["y_sw"] + m for m in range(ws.n_chunks)]
        t["ex_out"] = [torch.empty((ws.B, ws.S // ws.n_chunks, ws.T * ws.n_chunks, ws.C),
                                   dtype=torch.bfloat16, device=dev) for _ in range(ws.n_chunks)]
    if "switch_k3" in wanted:
        t["x_k3"] = t["x_sw"].view(ws.B, ws.T, 64, ws.S // 64, ws.C)
        t["y_k3"] = torch.empty((ws.n_chunks, ws.B, 64 // ws.n_chunks, ws.S // 64, ws.T, ws.C),
                                dtype=torch.bfloat16, device=dev)
    if "split" in wanted:
        t["y_split"] = torch.empty((ws.B, ws.T, ws.S // ws.n_chunks, ws.C), dtype=torch.bfloat16,
                                   device=dev)
    if "gather" in wanted:
        dsp.dsp_switch(t["x_sw"], 1, 2, ws.n_chunks, out=t["y_sw"])
        t["g_in"] = [t["y_sw"][m] for m in range(ws.n_chunks)]        # [B, S/8, T, C] each
        t["g_out"] = torch.empty((ws.B, ws.S // ws.n_chunks, ws.T * ws.n_chunks, ws.C),
                                 dtype=torch.bfloat16, device=dev)
    if "spatial" in wanted:
        t["q_sp"], t["k_sp"], t["v_sp"] = (to_dev(a, "bf16") for a in synth.qkv_inputs(wsp, "BTSC"))
        t["o_sp"] = torch.empty_like(t["q_sp"])
    if "temporal" in wanted:
        t["q_tp"], t["k_tp"], t["v_tp"] = (to_dev(a, "bf16") for a in synth.qkv_inputs(wtp, "BSTC"))
        t["o_tp"] = torch.empty_like(t["q_tp"])
    if "temporal_strided" in wanted:
        # the same tensors left in the unswitched (B, T, S, C) layout
        t["tq_tsc"] = [a.permute(0, 2, 1, 3).contiguous() for a in (t["q_tp"], t["k_tp"], t["v_tp"])]
        t["to_tsc"] = torch.empty_like(t["tq_tsc"][0])
    for kind in ("spatial", "temporal"):
        if f"attn_bwd_{kind}" in wanted:
            sfx = "sp" if kind == "spatial" else "tp"
            w = wsp if kind == "spatial" else wtp
            q = t[f"q_{sfx}"]
            gen = torch.Generator(device=dev).manual_seed(w.seed + 100)
            t[f"do_{sfx}"] = torch.randn(q.shape, generator=gen, device=dev).to(torch.bfloat16)
            t[f"of_{sfx}"], t[f"lse_{sfx}"] = dsp.dsp_attn_fwd_lse(q, t[f"k_{sfx}"], t[f"v_{sfx}"], w.H)
            t[f"g_{sfx}"] = [torch.empty_like(q) for _ in range(3)]
            t[f"dl_{sfx}"] = torch.empty(q.numel() // w.D, dtype=torch.float32, device=dev)
    if "block" in wanted:
        x_bl_np, p_bl = synth.block_inputs(wbl)
        t["x_bl"] = to_dev(x_bl_np, "f32")
        t["w_bl"] = {n: (None if v is None else to_dev(v, "bf16")) for n, v in p_bl.items()}
        t["y_bl"] = torch.empty((wbl.B, wbl.S, wbl.T, wbl.C), dtype=torch.float32, device=dev)
        ws_bytes = dsp.block_workspace_bytes(wbl.B, wbl.T, wbl.S, wbl.C, wbl.H, wbl.F, dsp.DSP_BF16)
        t["ws_bl"] = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
        del x_bl_np, p_bl
    if wanted & {"block_train_fwd", "block_bwd"}:
        gen = torch.Generator(device=dev).manual_seed(wbl.seed + 100)
        t["dy_bl"] = torch.randn((wbl.B, wbl.S, wbl.T, wbl.C), generator=gen, device=dev)
        t["y_tr"], t["sv_bl"] = dsp.dsp_st_block_forward_train(t["x_bl"], t["w_bl"], wbl.H)
        t["dx_bl"], t["g_bl"] = dsp.dsp_st_block_backward(t["x_bl"], t["dy_bl"], t["w_bl"], t["sv_bl"], wbl.H)
        t["bws_bl"] = torch.empty(int(dsp.lib().dsp_st_block_backward_workspace_bytes(
            wbl.B, wbl.T, wbl.S, wbl.C, wbl.H, wbl.F, dsp.DSP_BF16)), dtype=torch.uint8, device=dev)
    # the tiny fp32 chain (launch-latency bound): eager calls and a captured HIP graph
    wtc = W["tiny_chain_f32"]
    x_tc, p_tc = synth.chain_inputs(wtc)
    t["x_tc"] = to_dev(x_tc, "f32")
    t["w_tc"] = {n: to_dev(v, "f32") for n, v in p_tc.items()}
    t["y_tc"] = torch.empty((wtc.B, wtc.S, wtc.T, wtc.C), dtype=torch.float32, device=dev)
    t["ws_tc"] = torch.empty(dsp.block_workspace_bytes(wtc.B, wtc.T, wtc.S, wtc.C, wtc.H, 0, dsp.DSP_F32),
                             dtype=torch.uint8, device=dev)

    def run_tiny():
        dsp.dsp_st_block_forward(t["x_tc"], t["w_tc"], wtc.H, flags=dsp.DSP_BLOCK_ATTN_ONLY, out=t["y_tc"],
                                 workspace=t["ws_tc"])

    side = torch.cuda.Stream()
    side.wait_stream(stream)
    with torch.cuda.stream(side):
        run_tiny()
    stream.wait_stream(side)
    torch.cuda.synchronize()
    tiny_graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(tiny_graph):
        run_tiny()
    torch.cuda.synchronize()

    def run_switch():
        dsp.dsp_switch(t["x_sw"], 1, 2, ws.n_chunks, out=t["y_sw"])

    def run_switch_inv():
        dsp.dsp_switch(t["x_inv"], 1, 2, ws.n_chunks, out=t["y_inv"])

    def run_exchange():
        dsp.dsp_exchange_unpack(t["ex_in"], out=t["ex_out"])

    def run_temporal_strided():
        v = [a.permute(0, 2, 1, 3) for a in t["tq_tsc"]]
        dsp.dsp_attn_strided(*v, wtp.H, out=t["to_tsc"].permute(0, 2, 1, 3))

    def run_switch_k3():
        dsp.dsp_switch(t["x_k3"], 1, 2, ws.n_chunks, out=t["y_k3"])

    def run_split():
        dsp.dsp_split(t["x_sw"], 2, ws.n_chunks, 3, out=t["y_split"])

    def run_gather():
        dsp.dsp_gather(t["g_in"], 2, out=t["g_out"])

    def run_spatial():
        dsp.dsp_spatial_attn(t["q_sp"], t["k_sp"], t["v_sp"], wsp.H, out=t["o_sp"])

    def run_temporal():
        dsp.dsp_temporal_attn(t["q_tp"], t["k_tp"], t["v_tp"], wtp.H, out=t["o_tp"])

    def run_block():
        dsp.dsp_st_block_forward(t["x_bl"], t["w_bl"], wbl.H, out=t["y_bl"], workspace=t["ws_bl"])

    def run_bwd(sfx, w):
        dsp.dsp_attn_bwd(t[f"q_{sfx}"], t[f"k_{sfx}"], t[f"v_{sfx}"], t[f"of_{sfx}"], t[f"do_{sfx}"],
                         t[f"lse_{sfx}"], w.H, *t[f"g_{sfx}"], delta=t[f"dl_{sfx}"])

    def run_attn_bwd_spatial():
        run_bwd("sp", wsp)

    def run_attn_bwd_temporal():
        run_bwd("tp", wtp)

    def run_block_train_fwd():
        dsp.dsp_st_block_forward_train(t["x_bl"], t["w_bl"], wbl.H, out=t["y_tr"], saved=t["sv_bl"])

    def run_block_bwd():
        dsp.dsp_st_block_backward(t["x_bl"], t["dy_bl"], t["w_bl"], t["sv_bl"], wbl.H, dx=t["dx_bl"],
                                  grads=t["g_bl"], workspace=t["bws_bl"])

    def run_copy():
        dsp.dsp_switch(t["x_sw"], 1, 1, 1, out=t["y_sw"].view(t["x_sw"].shape))

    probe_ws = torch.empty(dsp.probe_mfma_workspace_bytes(), dtype=torch.uint8, device=dev)

    def run_tiny_graph():
        tiny_graph.replay()

    def run_mfma_probe():
        dsp.dsp_probe_mfma(PROBE_ITERS, probe_ws)

    parts = [("switch", run_switch), ("switch_inv", run_switch_inv), ("spatial", run_spatial),
             ("temporal", run_temporal), ("block", run_block)]
    # timed on its own after the steps: not a step of the single-GPU hot path
    extras = [("exchange", run_exchange), ("temporal_strided", run_temporal_strided),
              ("switch_k3", run_switch_k3), ("split", run_split), ("gather", run_gather),
              ("attn_bwd_spatial", run_attn_bwd_spatial), ("attn_bwd_temporal", run_attn_bwd_temporal),
              ("block_train_fwd", run_block_train_fwd), ("block_bwd", run_block_bwd),
              ("mfma_probe", run_mfma_probe), ("tiny_chain", run_tiny), ("tiny_chain_graph", run_tiny_graph)]
    if args.only:
        every = dict(parts + extras)
        parts, extras = [(args.only, run_copy if args.only == "copy" else every[args.only])], []

    for _ in range(args.warmup):
        for _, fn in parts:
            fn()
    torch.cuda.synchronize()

    K = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(parts) + 1)] for _ in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(K):
        ev[s][0].record(stream)
        for i, (_, fn) in enumerate(parts):
            fn()
            ev[s][i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    samples = {name: [ev[s][i].elapsed_time(ev[s][i + 1]) for s in range(K)] for i, (name, _) in enumerate(parts)}
    for name, fn in extras:
        for _ in range(args.warmup):
            fn()
        xev = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
        torch.cuda.synchronize()
        xev[0].record(stream)
        for s in range(K):
            fn()
            xev[s + 1].record(stream)
        torch.cuda.synchronize()
        samples[name] = [xev[s].elapsed_time(xev[s + 1]) for s in range(K)]
    ms = {name: float(np.mean(v)) for name, v in samples.items()}
    ms_median = {name: float(np.median(v)) for name, v in samples.items()}
    ms_min = {name: float(np.min(v)) for name, v in samples.items()}
    if args.only:
        print(json.dumps({"only": args.only, "steps": K, "kernel_ms": ms}), flush=True)
        return

    # the practical HBM ceiling of a streaming copy: a device-to-device copy of
    # the 604 MB switch tensor (torch copy_, one call per event pair)
    d2d = None
    if "switch" in wanted:
        dst = torch.empty_like(t["x_sw"])
        for _ in range(args.warmup):
            dst.copy_(t["x_sw"])
        cev = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
        torch.cuda.synchronize()
        cev[0].record(stream)
        for s_ in range(K):
            dst.copy_(t["x_sw"])
            cev[s_ + 1].record(stream)
        torch.cuda.synchronize()
        cs = [cev[i].elapsed_time(cev[i + 1]) for i in range(K)]
        nb = 2.0 * t["x_sw"].numel() * t["x_sw"].element_size()
        d2d = {"bytes": int(nb), "GBps_median": round(nb / (np.median(cs) * 1e-3) / 1e9, 1),
               "GBps_max": round(nb / (np.min(cs) * 1e-3) / 1e9, 1)}
        del dst

    # ---- accounting
    sw_bytes = 2.0 * t["x_sw"].numel() * t["x_sw"].element_size()
    F_sp = attn_flops(wsp.B * wsp.T * wsp.H, wsp.S, wsp.D)
    F_tp = attn_flops(wtp.B * wtp.S * wtp.H, wtp.T, wtp.D)
    tp_bytes = 4.0 * t["q_tp"].numel() * 2
    tp_bytes_all = tp_bytes
    tok = wbl.B * wbl.T * wbl.S
    C, F = wbl.C, wbl.F
    F_gemm = 2.0 * tok * C * (3 * C) * 2 + 2.0 * tok * C * C * 2 + 2.0 * tok * C * F * 2
    F_att = attn_flops(wbl.B * wbl.T * wbl.H, wbl.S, wbl.D) + attn_flops(wbl.B * wbl.S * wbl.H, wbl.T, wbl.D)
    F_bl = F_gemm + F_att
    F_bl_bwd = 2.0 * F_gemm + 2.5 * F_att

    sp_tflops = F_sp / (ms["spatial"] * 1e-3) / 1e12
    tp_tflops = F_tp / (ms["temporal"] * 1e-3) / 1e12
    attn_tflops = (F_sp + F_tp) / ((ms["spatial"] + ms["temporal"]) * 1e-3) / 1e12
    sw_gbps = sw_bytes / (ms["switch"] * 1e-3) / 1e9
    sw_inv_gbps = sw_bytes / (ms["switch_inv"] * 1e-3) / 1e9
    ex_gbps = ws.n_chunks * sw_bytes / (ms["exchange"] * 1e-3) / 1e9
    tps_gbps = tp_bytes_all / (ms["temporal_strided"] * 1e-3) / 1e9
    tp_gbps = tp_bytes / (ms["temporal"] * 1e-3) / 1e9
    k3_gbps = sw_bytes / (ms["switch_k3"] * 1e-3) / 1e9
    split_gbps = sw_bytes / ws.n_chunks / (ms["split"] * 1e-3) / 1e9
    gather_gbps = sw_bytes / (ms["gather"] * 1e-3) / 1e9

    traffic = measured_traffic(args.traffic)
    mfma_sustained = dsp.probe_mfma_flops(PROBE_ITERS) / (ms["mfma_probe"] * 1e-3) / 1e12

    out = {
        "metric": METRIC,
        "value": round(attn_tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / K, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "dsp_switch 1x64x4096x1152 bf16 -> 8 chunks and its inverse 1x4096x64x1152 -> 8 "
                        "chunks; 8-rank exchange+unpack of such shards; the shard as 1x64x64x64x1152 "
                        "switched T->H (K=3); split along S / gather along T of 8 shards; spatial attn B2 T16 S4096 H16 D72; "
                        "temporal attn B2 S512 T128 H16 D72; ST block B1 T32 S1024 C1152 H16 F4608; "
                        "attention backward of the spatial and temporal workloads; training forward and "
                        "backward of the ST block; the tiny fp32 chain B1 T4 S16 C64 H4 D16 (eager and "
                        "HIP-graph replay, us per call)",
            "attn_frac_mfma_peak": round(attn_tflops / MFMA_BF16_PEAK_TFLOPS, 4),
            "switch_GBps": round(sw_gbps, 1),
            "switch_frac_hbm_peak": round(sw_gbps / HBM_PEAK_GBPS, 4),
            "switch_inverse_GBps": round(sw_inv_gbps, 1),
            "switch_inverse_frac_hbm_peak": round(sw_inv_gbps / HBM_PEAK_GBPS, 4),
            "exchange_unpack_GBps": round(ex_gbps, 1),
            "exchange_unpack_frac_hbm_peak": round(ex_gbps / HBM_PEAK_GBPS, 4),
            "temporal_unswitched_layout_GBps": round(tps_gbps, 1),
            "switch_k3_GBps": round(k3_gbps, 1),
            "split_GBps": round(split_gbps, 1),
            "gather_GBps": round(gather_gbps, 1),
            "spatial_TFLOPs": round(sp_tflops, 2),
            "temporal_TFLOPs": round(tp_tflops, 2),
            "temporal_GBps": round(tp_gbps, 1),
            "temporal_frac_hbm_peak": round(tp_gbps / HBM_PEAK_GBPS, 4),
            "block_TFLOPs": round(F_bl / (ms["block"] * 1e-3) / 1e12, 2),
            "attn_bwd_spatial_TFLOPs": round(2.5 * F_sp / (ms["attn_bwd_spatial"] * 1e-3) / 1e12, 2),
            "attn_bwd_temporal_TFLOPs": round(2.5 * F_tp / (ms["attn_bwd_temporal"] * 1e-3) / 1e12, 2),
            "block_train_fwd_TFLOPs": round(F_bl / (ms["block_train_fwd"] * 1e-3) / 1e12, 2),
            "block_bwd_TFLOPs": round(F_bl_bwd / (ms["block_bwd"] * 1e-3) / 1e12, 2),
            "tiny_chain_us": round(ms["tiny_chain"] * 1e3, 2),
            "tiny_chain_graph_us": round(ms["tiny_chain_graph"] * 1e3, 2),
            "kernel_ms": {k: round(v, 4) for k, v in ms.items()},
            "kernel_ms_median": {k: round(v, 4) for k, v in ms_median.items()},
            "kernel_ms_min": {k: round(v, 4) for k, v in ms_min.items()},
            "d2d_copy": d2d,
            "switch_frac_of_d2d_copy": round(sw_gbps / d2d["GBps_median"], 4) if d2d else None,
            "clocks": gpu_clocks(),
        },
        "roofline": {
            "kernel": "spatial attention attn_fwd_kernel<72,8,2,64,2,2> (B2 T16 S4096 H16 D72)",
            "bound": "mfma",
            "achieved": round(sp_tflops, 2),
            "peak": MFMA_BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(sp_tflops / MFMA_BF16_PEAK_TFLOPS, 4),
            "traffic": traffic,
        },
    }
    # context for roofline.frac: the bf16 MFMA rate this GPU sustains with every
    # CU busy (independent MFMA chains only), measured in this run
    out["mfma_sustained"] = {
        "value": round(mfma_sustained, 1),
        "unit": "TFLOP/s",
        "frac_of_peak": round(mfma_sustained / MFMA_BF16_PEAK_TFLOPS, 4),
        "spatial_frac_of_sustained": round(sp_tflops / mfma_sustained, 4),
        "how": "dsp_probe_mfma: 8 independent v_mfma_f32_32x32x16_bf16 chains per wave, 2 waves per SIMD, "
               "all CUs, operand bits changing every iteration; HIP events over %d launches" % K,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.cpu_budget)
    print(json.dumps(out), flush=True)


def gpu_clocks():
    """The current shader / memory / fabric clocks as rocm-smi reports them (a
    child process; None when the tool is not there or fails)."""
    import subprocess
    try:
        r = subprocess.run(["rocm-smi", "--showclocks", "--json"], capture_output=True, text=True, timeout=30)
        d = json.loads(r.stdout)
    except Exception:
        return None
    card = next(iter(d.values()), {}) if isinstance(d, dict) else {}
    return {k: v for k, v in card.items() if "clock" in k.lower() or "clk" in k.lower()} or None


def measured_traffic(path):
    """HBM bytes per launch of the spatial kernel from the committed counter
    summary, or None when the summary is missing or the kernel source has
    changed since the counters were taken."""
    import hashlib
    if not path or not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    src = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2403_10266_amd", "csrc",
                       "attn_bf16.hip")
    with open(src, "rb") as f:
        sha = hashlib.sha256(f.read()).hexdigest()[:16]
    if kv.get("spatial_source_sha256_16") != sha or "spatial_bytes_per_launch" not in kv:
        return None
    return int(kv["spatial_bytes_per_launch"])


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(budget_s: float) -> dict:
    """The fp64 oracle on this host's cores, on bounded samples of the same
    workloads (independent units, so throughput is per-unit exact): attention
    with BLAS threads equal to the CPUs this process may run on (capped by
    OMP_NUM_THREADS, the host's share per GPU), the same with one thread, and
    the switch oracle (a uint16 gather) on a slice of the switch shard."""
    import oracle
    import synth
    from threadpoolctl import threadpool_limits
    affinity = len(os.sched_getaffinity(0))
    threads = min(affinity, int(os.environ.get("OMP_NUM_THREADS", affinity) or affinity))
    W = synth.WORKLOADS
    wsp, wtp, wsw = W["spatial_bf16_B2_T16_S4096"], W["temporal_bf16_B2_S512_T128"], W["switch_bf16_T64_S4096"]
    D = wsp.D

    def unit_set(w, L, n):
        g = synth.rng(w.seed)
        return tuple(synth.bf16_round(synth.normal_f32(g, (n, L, D))).astype(np.float64) for _ in range(3))

    def attention_rate(budget, max_sp, max_tp):
        """(TFLOP/s, spatial units, temporal units, seconds, per-unit spatial times)"""
        t_sp = f_sp = 0.0
        n_sp = 0
        per_unit = []
        q, k, v = unit_set(wsp, wsp.S, 1)
        while t_sp < budget / 2 and n_sp < max_sp:
            t0 = time.perf_counter()
            oracle.attention(q[0], k[0], v[0])
            per_unit.append(time.perf_counter() - t0)
            t_sp += per_unit[-1]
            f_sp += attn_flops(1, wsp.S, D)
            n_sp += 1
        t_tp = f_tp = 0.0
        n_tp = 0
        q, k, v = unit_set(wtp, wtp.T, 256)
        while t_tp < budget / 2 and n_tp < max_tp:
            t0 = time.perf_counter()
            oracle.attention(q, k, v)
            t_tp += time.perf_counter() - t0
            f_tp += attn_flops(256, wtp.T, D)
            n_tp += 256
        return (f_sp + f_tp) / (t_sp + t_tp) / 1e12, n_sp, n_tp, t_sp + t_tp, per_unit

    with threadpool_limits(limits=threads):
        rate, n_sp, n_tp, secs, per_unit = attention_rate(0.6 * budget_s, 512, 16384)
    with threadpool_limits(limits=1):
        rate1, n_sp1, n_tp1, secs1, per_unit1 = attention_rate(0.25 * budget_s, 512, 16384)
    # the switch oracle on the first 8 of the shard's 64 frames (75.5 MB), T -> S into 8 chunks
    frames = 8
    # (the generator's first draws: the same values as those frames of the full shard)
    xb = synth.f32_to_bf16_bits(synth.activations(wsw, synth.rng(wsw.seed), (wsw.B, frames, wsw.S, wsw.C)))
    sw_times = []
    for _ in range(3):
        t0 = time.perf_counter()
        oracle.switch(xb, 1, 2, wsw.n_chunks)
        sw_times.append(time.perf_counter() - t0)
    sw_bytes = 2.0 * xb.nbytes
    del xb
    return {
        "value": round(rate, 6),
        "unit": "TFLOP/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"fp64 NumPy oracle attention, {threads} BLAS threads: {n_sp} of 512 spatial units (L=4096, D=72) "
                  f"and {n_tp} of 16384 temporal units (L=128, D=72), same 4*L^2*D accounting; {secs:.1f} s of "
                  f"host time",
        "cpu_model": cpu_model(),
        "affinity_cpus": affinity,
        "one_thread": {"value": round(rate1, 6), "unit": "TFLOP/s",
                       "sample": f"{n_sp1} spatial and {n_tp1} temporal units, {secs1:.1f} s"},
        "spatial_unit_s": {"median": round(float(np.median(per_unit)), 4), "min": round(float(np.min(per_unit)), 4),
                           "one_thread_median": round(float(np.median(per_unit1)), 4)},
        "switch": {"GBps_median": round(sw_bytes / np.median(sw_times) / 1e9, 3),
                   "GBps_max": round(sw_bytes / np.min(sw_times) / 1e9, 3),
                   "sample": f"oracle.switch (uint16 gather, single-threaded NumPy) of frames 0-{frames - 1} of the "
                             f"1x64x4096x1152 shard, T -> S into 8 chunks, {sw_bytes / 1e6:.0f} MB moved, 3 runs"},
    }


if __name__ == "__main__":
    main()
