"""Benchmark of the whole hot path on one MI355X.

A step runs every part of the path once, on seeded synthetic inputs already resident in
HBM:
  * bf16 GEMM 8192 x 8192 x 8192, bf16 and fp32 outputs
  * bf16 GEMM M=8192 N=1024 K=16384, bf16 and fp32 outputs
  * skinny GEMM 4096 x 32 x 4096, bf16 and fp32 inputs (fp32 out); also N = 1 (bf16)
  * GRU forward T=64, batch 32, input = hidden = 1024, bf16 weights (also T=128 and batch 4)
  * separable depthwise conv 32 x 56 x 56 x 128 -> 256, bf16 (fp32 out) and fp32
  * 1D convolution 32 sequences x 1024 positions, 512 -> 512 channels, 5 taps, bf16 (fp32 out)
  * fp32 GEMM 128^3; as context, fp32 GEMM 4096^3 (run as six bf16 term products)
Each part is bracketed by HIP events on the stream the library launches on (torch's current
stream), so the per-part times are device times; after the timed steps each part also runs
alone, calls queued back to back between two events ("us_b2b": device time per call without
the per-call event and launch gaps, which dominate the small parts).  The HBM-bound parts (skinny GEMM, GRU,
separable conv) rotate over enough input copies that every call reads from HBM rather than
the 256 MB memory-side cache; the same call on one warm buffer set is reported beside it as
"<name>_mall_warm".  `value` is the GEMM throughput of the
large bf16 GEMMs (total FLOP / total time); GRU timesteps/s, separable-conv GB/s and the
rest are reported under "components".  `roofline` covers the dominant kernel (the square
bf16 GEMM, bf16 output); `cpu_baseline` times the CPU oracle on a bounded sample.

After the timing, every configuration runs once more and is compared with the CPU oracle
("parity": maximum normalised error, tolerance, pass/fail, oracle seconds and threads).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline] [--no-parity]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "GEMM TFLOP/s (% of MFMA peak); GRU timesteps/sec; dwsep conv GB/s"
PEAK_BF16_TFLOPS = 2516.6
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBPS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-parity", action="store_true", help="skip the per-configuration check against the oracle")
    ap.add_argument("--only", default="", help="comma list of component names to run (profiling)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="time plain device copies / fills of known size (HBM reference, counter scaling)")
    return ap.parse_args()


def copy_calibration():
    """Plain torch copies and fills of 256 MiB and 1 GiB: the achieved HBM rate of trivial
    streaming kernels on this device, and the reference the FETCH_SIZE / WRITE_SIZE counters
    are scaled by (each copy reads and writes exactly its size)."""
    import torch
    dev = torch.device("cuda:0")
    out = {}
    for mib in (256, 1024):
        n = mib * (1 << 20) // 4
        a = torch.ones(n, device=dev)
        b = torch.empty(n, device=dev)
        for _ in range(3):
            b.copy_(a)
            b.fill_(2.0)
        torch.cuda.synchronize()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        R = 10
        e[0].record()
        for _ in range(R):
            b.copy_(a)
        e[1].record()
        for _ in range(R):
            b.fill_(3.0)
        e[2].record()
        torch.cuda.synchronize()
        tc = e[0].elapsed_time(e[1]) / R * 1e-3
        tf = e[1].elapsed_time(e[2]) / R * 1e-3
        out[f"copy_{mib}MiB"] = {"us": round(tc * 1e6, 1), "GB/s": round(2 * n * 4 / tc / 1e9, 1)}
        out[f"fill_{mib}MiB"] = {"us": round(tf * 1e6, 1), "GB/s": round(n * 4 / tf / 1e9, 1)}
    print(json.dumps({"copy_calibration": out}), flush=True)


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on exactly one GPU: this library has no multi-GPU path "
              "(the kernels are timed on one GPU's share of the work).", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_1810_09958_amd as isam
    import synth
    from synth import workloads

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    def gpu(a):
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    t_setup = time.time()
    only = set(s for s in args.only.split(",") if s)
    comps = []   # (name, callable, info dict)

    def want(name):
        return not only or name in only

    # -- large bf16 GEMMs -------------------------------------------------------------
    sq = workloads.gemm_square_bf16()
    Aq, Bq = gpu(sq["A_bf16"]), gpu(sq["B_bf16"])
    del sq
    Cq16 = torch.empty((8192, 8192), device=dev, dtype=torch.bfloat16)
    Cq32 = torch.empty((8192, 8192), device=dev, dtype=torch.float32)
    rc = workloads.gemm_rect_bf16()
    Ar, Br = gpu(rc["A_bf16"]), gpu(rc["B_bf16"])
    del rc
    Cr16 = torch.empty((8192, 1024), device=dev, dtype=torch.bfloat16)
    Cr32 = torch.empty((8192, 1024), device=dev, dtype=torch.float32)
    f_sq = 2.0 * 8192 ** 3
    f_rc = 2.0 * 8192 * 1024 * 16384

    def gemm_bytes(M, N, K, cbytes):
        return 2 * (M * K + K * N) + cbytes * M * N

    for name, A, B, C, fl, M, N, K in [
        ("gemm_8192x8192x8192_bf16_out_bf16", Aq, Bq, Cq16, f_sq, 8192, 8192, 8192),
        ("gemm_8192x8192x8192_bf16_out_f32", Aq, Bq, Cq32, f_sq, 8192, 8192, 8192),
        ("gemm_8192x1024x16384_bf16_out_bf16", Ar, Br, Cr16, f_rc, 8192, 1024, 16384),
        ("gemm_8192x1024x16384_bf16_out_f32", Ar, Br, Cr32, f_rc, 8192, 1024, 16384),
    ]:
        ws = torch.empty(max(1, isam.gemm_workspace_size(M, N, K, 1, 1 if C.dtype == torch.bfloat16 else 0)),
                         device=dev, dtype=torch.uint8)
        if want(name):
            comps.append((name, (lambda A=A, B=B, C=C, ws=ws: isam.gemm(A, B, C, workspace=ws)),
                          {"kind": "gemm_bf16", "flop": fl,
                           "bytes": gemm_bytes(M, N, K, C.element_size())}))

    # The HBM-bound parts (skinny GEMM, GRU, separable conv) have working sets that fit the
    # 256 MB memory-side cache.  Their reported numbers rotate over enough copies of the
    # inputs (and large outputs) that one pass over the rotation set exceeds 2 x 256 MB, so
    # every call reads from HBM; the same call on one buffer set is reported beside it as
    # "<name>_mall_warm".
    ROTATE_BYTES = 2 * 256 * (1 << 20)

    def n_sets(bytes_per_set):
        return max(2, -(-ROTATE_BYTES // bytes_per_set) + 1)

    def add_rotated(name, make_call, sets, info):
        """make_call(i) -> the call on buffer set i; adds the rotated and the MALL-warm entry."""
        calls = [make_call(i) for i in range(sets)]
        state = {"i": 0}

        def rotated():
            calls[state["i"]]()
            state["i"] = (state["i"] + 1) % len(calls)

        comps.append((name, rotated, dict(info, rotation_sets=sets)))
        # MALL-warm: the same call on set 0, right after an untimed call on set 0.
        comps.append((name + "_mall_warm", calls[0], dict(info, rotation_sets=1, pre=calls[0])))

    # -- skinny GEMM ------------------------------------------------------------------
    sk = workloads.skinny()
    for name, A_h, B_h, es in [("skinny_4096x32x4096_bf16", sk["A_bf16"], sk["B_bf16"], 2),
                               ("skinny_4096x32x4096_f32", sk["A"], sk["B"], 4)]:
        if not want(name):
            continue
        A0, B0 = gpu(A_h), gpu(B_h)
        sets = n_sets(A0.numel() * es)
        As = [A0] + [A0.clone() for _ in range(sets - 1)]
        Bs = [B0] + [B0.clone() for _ in range(sets - 1)]
        Cs = [torch.empty((4096, 32), device=dev, dtype=torch.float32) for _ in range(sets)]
        ws = torch.empty(max(1, isam.gemm_workspace_size(4096, 32, 4096, 1 if es == 2 else 0, 0)),
                         device=dev, dtype=torch.uint8)
        add_rotated(name, lambda i, As=As, Bs=Bs, Cs=Cs, ws=ws: (lambda: isam.gemm(As[i], Bs[i], Cs[i], workspace=ws)),
                    sets, {"kind": "skinny", "flop": 2.0 * 4096 * 32 * 4096,
                           "bytes": es * (4096 * 4096 + 4096 * 32) + 4 * 4096 * 32})
    # narrow product (batch 1, matrix-vector), context point: dot-product kernel
    if want("gemv_4096x1x4096_bf16"):
        A0, B0 = gpu(sk["A_bf16"]), gpu(np.ascontiguousarray(sk["B_bf16"][:, :1]))
        sets = n_sets(A0.numel() * 2)
        As = [A0] + [A0.clone() for _ in range(sets - 1)]
        Cs = [torch.empty((4096, 1), device=dev, dtype=torch.float32) for _ in range(sets)]
        ws = torch.empty(1, device=dev, dtype=torch.uint8)
        add_rotated("gemv_4096x1x4096_bf16", lambda i, As=As, Cs=Cs, B0=B0, ws=ws: (lambda: isam.gemm(As[i], B0, Cs[i], workspace=ws)),
                    sets, {"kind": "skinny", "flop": 2.0 * 4096 * 4096,
                           "bytes": 2 * (4096 * 4096 + 4096) + 4 * 4096})
    del sk

    # -- GRU --------------------------------------------------------------------------
    T, Bt, I, H = 64, 32, 1024, 1024
    if want("gru_T64_B32_H1024_bf16"):
        g = workloads.gru()
        gx, gW, gU, gb = gpu(g["x_bf16"]), gpu(g["W_bf16"]), gpu(g["U_bf16"]), gpu(g["bias"])
        del g
        sets = n_sets(2 * (T * Bt * I + 6 * H * I) + 4 * T * Bt * H)
        gsets = [(gx, gW, gU)] + [(gx.clone(), gW.clone(), gU.clone()) for _ in range(sets - 1)]
        hseqs = [torch.empty((T, Bt, H), device=dev) for _ in range(sets)]
        g_hT = torch.empty((Bt, H), device=dev)
        g_ws = torch.empty(isam.gru_forward_workspace_size(T, Bt, I, H, 1), device=dev, dtype=torch.uint8)
        add_rotated("gru_T64_B32_H1024_bf16",
                    lambda i: (lambda: isam.gru_forward(gsets[i][0], gsets[i][1], gsets[i][2], bias=gb,
                                                        h_seq=hseqs[i], h_T=g_hT, workspace=g_ws)),
                    sets, {"kind": "gru", "steps": T,
                           "flop": 2.0 * T * Bt * 3 * H * (I + H),
                           "bytes": 2 * (3 * H * I + 3 * H * H + T * Bt * I) + 4 * T * Bt * H})

        # the same call (MALL-warm, one buffer set) under the persistent schedule
        comps.append(("gru_T64_B32_H1024_bf16_persistent_mall_warm",
                      (lambda: isam.gru_forward(gsets[0][0], gsets[0][1], gsets[0][2], bias=gb,
                                                h_seq=hseqs[0], h_T=g_hT, workspace=g_ws)),
                      {"kind": "gru", "steps": T, "env": {"ISAM_GRU_MODE": "persistent"},
                       "flop": 2.0 * T * Bt * 3 * H * (I + H),
                       "bytes": 2 * (3 * H * I + 3 * H * H + T * Bt * I) + 4 * T * Bt * H}))

    # GRU variants (context points): the paper's 128 steps; a small batch.
    for (gT, gB, gname) in [(128, 32, "gru_T128_B32_H1024_bf16"), (64, 4, "gru_T64_B4_H1024_bf16")]:
        if not want(gname):
            continue
        g = workloads.gru(T=gT, batch=gB)
        vx, vW, vU, vb = gpu(g["x_bf16"]), gpu(g["W_bf16"]), gpu(g["U_bf16"]), gpu(g["bias"])
        del g
        vh = torch.empty((gT, gB, H), device=dev)
        vT = torch.empty((gB, H), device=dev)
        vws = torch.empty(isam.gru_forward_workspace_size(gT, gB, I, H, 1), device=dev, dtype=torch.uint8)
        comps.append((gname, (lambda vx=vx, vW=vW, vU=vU, vb=vb, vh=vh, vT=vT, vws=vws:
                              isam.gru_forward(vx, vW, vU, bias=vb, h_seq=vh, h_T=vT, workspace=vws)),
                      {"kind": "gru", "steps": gT, "flop": 2.0 * gT * gB * 3 * H * (I + H),
                       "bytes": 2 * (3 * H * I + 3 * H * H + gT * gB * I) + 4 * gT * gB * H}))

    # -- separable depthwise conv -------------------------------------------------------
    d = workloads.dwsep()
    for name, X_h, D_h, P_h, es, oes in [
            ("dwsep_32x56x56x128_256_bf16_out_f32", d["X_bf16"], d["D_bf16"], d["P_bf16"], 2, 4),
            ("dwsep_32x56x56x128_256_bf16_out_bf16", d["X_bf16"], d["D_bf16"], d["P_bf16"], 2, 2),
            ("dwsep_32x56x56x128_256_f32", d["X"], d["D"], d["P"], 4, 4)]:
        if not want(name):
            continue
        X0, Dw, P = gpu(X_h), gpu(D_h), gpu(P_h)
        sets = n_sets(X0.numel() * es + oes * 100352 * 256)
        Xs = [X0] + [X0.clone() for _ in range(sets - 1)]
        ys = [torch.empty((32, 56, 56, 256), device=dev, dtype=torch.float32 if oes == 4 else torch.bfloat16)
              for _ in range(sets)]
        it = 1 if es == 2 else 0
        ot = 0 if oes == 4 else 1
        ws = torch.empty(isam.dwsep_conv_workspace_size(32, 56, 56, 128, 1, 3, 3, 1, 1, 256, it, ot),
                         device=dev, dtype=torch.uint8)
        add_rotated(name, lambda i, Xs=Xs, Dw=Dw, P=P, ys=ys, ws=ws: (lambda: isam.dwsep_conv(Xs[i], Dw, P, out=ys[i], workspace=ws)),
                    sets, {"kind": "dwsep", "flop": 2.0 * 100352 * (9 * 128 + 128 * 256),
                           # fused minimum: X read once, y written once (+ the small filters)
                           "bytes": es * (32 * 56 * 56 * 128 + 9 * 128 + 128 * 256) + oes * 100352 * 256})
    # The same convolution unfused (depthwise kernel writes Y, then the pointwise GEMM reads it):
    # times the standalone depthwise stencil and the pointwise product as separate launches.
    if want("dwsep_32x56x56x128_256_bf16_out_bf16_unfused"):
        X0, Dw, P = gpu(d["X_bf16"]), gpu(d["D_bf16"]), gpu(d["P_bf16"])
        sets = n_sets(2 * (3 * 32 * 56 * 56 * 128 + 100352 * 256))
        Xs = [X0] + [X0.clone() for _ in range(sets - 1)]
        ys = [torch.empty((32, 56, 56, 256), device=dev, dtype=torch.bfloat16) for _ in range(sets)]
        os.environ["ISAM_DWSEP_FUSED"] = "0"   # size of the unfused path: Y in the workspace
        wsu_bytes = isam.dwsep_conv_workspace_size(32, 56, 56, 128, 1, 3, 3, 1, 1, 256, 1, 1)
        del os.environ["ISAM_DWSEP_FUSED"]
        wsu = [torch.empty(wsu_bytes, device=dev, dtype=torch.uint8) for _ in range(sets)]
        add_rotated("dwsep_32x56x56x128_256_bf16_out_bf16_unfused",
                    lambda i, Xs=Xs, Dw=Dw, P=P, ys=ys, wsu=wsu: (lambda: isam.dwsep_conv(Xs[i], Dw, P, out=ys[i], workspace=wsu[i])),
                    sets, {"kind": "dwsep", "flop": 2.0 * 100352 * (9 * 128 + 128 * 256),
                           "env": {"ISAM_DWSEP_FUSED": "0"},
                           # X read, Y written and read back, y written (+ the small filters)
                           "bytes": 2 * (3 * 32 * 56 * 56 * 128 + 9 * 128 + 128 * 256) + 2 * 100352 * 256})
    del d

    # -- 1D convolution (second listing) as implicit GEMM --------------------------------
    if want("conv1d_32x1024_512x5x512_bf16"):
        w = workloads.conv1d()
        cA, cB = gpu(w["A_bf16"]), gpu(w["B_bf16"])
        del w
        cC = torch.empty((32, 1024, 512), device=dev, dtype=torch.float32)
        comps.append(("conv1d_32x1024_512x5x512_bf16", lambda: isam.conv1d(cA, cB, out=cC),
                      {"kind": "gemm_bf16_ctx", "flop": 2.0 * 32 * 1024 * 512 * 5 * 512,
                       "bytes": 2 * (32 * 1028 * 512 + 5 * 512 * 512) + 4 * 32 * 1024 * 512}))

    # -- small fp32 GEMM ------------------------------------------------------------------
    s1 = workloads.gemm_small_fp32()
    A1, B1 = gpu(s1["A"]), gpu(s1["B"])
    C1 = torch.empty((128, 128), device=dev)
    ws1 = torch.empty(max(1, isam.gemm_workspace_size(128, 128, 128, 0, 0)), device=dev, dtype=torch.uint8)
    if want("gemm_128x128x128_f32"):
        comps.append(("gemm_128x128x128_f32", lambda: isam.gemm(A1, B1, C1, workspace=ws1),
                      {"kind": "gemm_f32", "flop": 2.0 * 128 ** 3, "bytes": 3 * 4 * 128 * 128}))
    # -- large fp32 GEMM (context): the bf16-term split path ------------------------------
    if want("gemm_4096x4096x4096_f32_ctx"):
        A4 = gpu(synth.uniform(4096, 60, (4096, 4096), -1, 1))
        B4 = gpu(synth.uniform(4096, 61, (4096, 4096), -1, 1))
        C4 = torch.empty((4096, 4096), device=dev)
        ws4 = torch.empty(max(1, isam.gemm_workspace_size(4096, 4096, 4096, 0, 0)), device=dev, dtype=torch.uint8)
        comps.append(("gemm_4096x4096x4096_f32_ctx", lambda: isam.gemm(A4, B4, C4, workspace=ws4),
                      {"kind": "gemm_f32_split", "flop": 2.0 * 4096 ** 3, "bytes": 3 * 4 * 4096 * 4096}))
    torch.cuda.synchronize()
    t_setup = time.time() - t_setup

    stream = torch.cuda.current_stream()

    def run_step(evs=None):
        for i, (_, fn, info) in enumerate(comps):
            saved = {k: os.environ.get(k) for k in info.get("env", {})}
            os.environ.update(info.get("env", {}))
            if info.get("pre") is not None:
                info["pre"]()
            if evs is not None:
                evs[i][0].record(stream)
            fn()
            if evs is not None:
                evs[i][1].record(stream)
            for k, v in saved.items():
                if v is None:
                    os.environ.pop(k, None)
                else:
                    os.environ[k] = v

    for _ in range(args.warmup):
        run_step()
    torch.cuda.synchronize()

    K = args.steps
    events = [[[torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)]
               for _ in comps] for _ in range(K)]
    t0 = time.perf_counter()
    for k in range(K):
        run_step(events[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    # Back to back: each part alone, R calls queued between two events (rotated parts keep
    # rotating), so the figure is the device time per call without the per-call event and
    # launch gaps of the step -- the rate a stream of such calls sustains.
    b2b = {}
    for i, (name, fn, info) in enumerate(comps):
        saved = {k: os.environ.get(k) for k in info.get("env", {})}
        os.environ.update(info.get("env", {}))
        per_call_s = max(1e-6, float(np.mean([events[k][i][0].elapsed_time(events[k][i][1]) for k in range(K)])) * 1e-3)
        R = int(min(200, max(10, 5e-3 / per_call_s)))
        fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(R):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        b2b[name] = (e0.elapsed_time(e1) * 1e3 / R, R)
        for k, v in saved.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v

    results = {}
    for i, (name, _, info) in enumerate(comps):
        ms = [events[k][i][0].elapsed_time(events[k][i][1]) for k in range(K)]
        avg = float(np.mean(ms))
        r = {"us_avg": round(avg * 1e3, 2), "us_median": round(float(np.median(ms)) * 1e3, 2),
             "us_p10": round(float(np.percentile(ms, 10)) * 1e3, 2),
             "us_p90": round(float(np.percentile(ms, 90)) * 1e3, 2)}
        s = avg * 1e-3
        tfl = info["flop"] / s / 1e12
        gbs = info["bytes"] / s / 1e9
        r["TFLOP/s"] = round(tfl, 2)
        r["GB/s"] = round(gbs, 1)
        if info["kind"] in ("gemm_bf16", "gemm_bf16_ctx"):
            r["frac_bf16_peak"] = round(tfl / PEAK_BF16_TFLOPS, 4)
        elif info["kind"] == "gemm_f32":
            r["frac_f32_peak"] = round(tfl / PEAK_F32_TFLOPS, 6)
        elif info["kind"] == "gemm_f32_split":
            # six bf16 products per fp32 product on the bf16 matrix cores
            r["frac_bf16_peak_of_term_products"] = round(6 * tfl / PEAK_BF16_TFLOPS, 4)
        elif info["kind"] in ("skinny", "dwsep"):
            r["frac_hbm_peak"] = round(gbs / PEAK_HBM_GBPS, 4)
        us_b, R = b2b[name]
        r["us_b2b"] = round(us_b, 2)
        r["b2b_calls"] = R
        if info["kind"] in ("gemm_bf16", "gemm_bf16_ctx"):
            r["frac_bf16_peak_b2b"] = round(info["flop"] / (us_b * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, 4)
        elif info["kind"] in ("skinny", "dwsep"):
            r["frac_hbm_peak_b2b"] = round(info["bytes"] / (us_b * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4)
        elif info["kind"] == "gru":
            r["timesteps_per_s_b2b"] = round(info["steps"] / (us_b * 1e-6), 1)
        if info.get("rotation_sets", 1) > 1:
            r["rotation_sets"] = info["rotation_sets"]
        if info["kind"] == "gru":
            r["timesteps_per_s"] = round(info["steps"] / s, 1)
            r["us_per_timestep"] = round(avg * 1e3 / info["steps"], 3)
        results[name] = r

    gemm_names = [n for n, _, i in comps if i["kind"] == "gemm_bf16"]
    if gemm_names:
        tot_flop = sum(i["flop"] for n, _, i in comps if i["kind"] == "gemm_bf16")
        tot_s = sum(results[n]["us_avg"] for n in gemm_names) * 1e-6
        value = tot_flop / tot_s / 1e12
    else:
        value = None

    out = {
        "metric": METRIC,
        "value": round(value, 2) if value is not None else None,
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
            "workload": "hot path: bf16 GEMM 8192^3 + 8192x1024x16384 (bf16/fp32 out), skinny 4096x32x4096, "
                        "GRU T64 B32 I1024 H1024, dwsep 32x56x56x128->256, fp32 GEMM 128^3",
            "value_is": "large bf16 GEMM throughput (total FLOP / total device time of those launches)",
            "parallelism": "single GPU",
        },
    }
    if value is not None:
        out["frac_of_bf16_peak"] = round(value / PEAK_BF16_TFLOPS, 4)
    dom = "gemm_8192x8192x8192_bf16_out_bf16"
    if dom in results:
        ach = results[dom]["TFLOP/s"]
        traffic = measured_traffic("gemm_dma_256x256_bf16_8192cubed_traffic.json")
        out["roofline"] = {"kernel": "gemm_dma_kernel<256, 256, false, 2, 4, true, false> (8192^3, bf16 out)",
                           "bound": "mfma", "achieved": ach, "peak": PEAK_BF16_TFLOPS,
                           "unit": "TFLOP/s", "frac": round(ach / PEAK_BF16_TFLOPS, 4),
                           "traffic": traffic}
        if traffic is not None:
            out["roofline"]["traffic_unit"] = "bytes per launch (HBM-side, rocprofv3 FETCH_SIZE/WRITE_SIZE, copy-scaled)"
            out["roofline"]["traffic_GBps"] = round(traffic / (results[dom]["us_avg"] * 1e-6) / 1e9, 1)
    if "gru_T64_B32_H1024_bf16" in results:
        out["gru_timesteps_per_s"] = results["gru_T64_B32_H1024_bf16"]["timesteps_per_s"]
    if "dwsep_32x56x56x128_256_bf16_out_f32" in results:
        out["dwsep_GBps"] = results["dwsep_32x56x56x128_256_bf16_out_f32"]["GB/s"]
    out["components"] = results
    out["setup_s"] = round(t_setup, 1)

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline()
    if not args.no_parity:
        out["parity"] = parity_per_config(isam, gpu)
    print(json.dumps(out), flush=True)


def parity_per_config(isam, gpu):
    """Each benchmark configuration once more through the library (the same launch
    configuration the timing uses), against the CPU oracle: maximum normalised error
    (|gpu - oracle| / sum|a||b|; for the GRU the absolute error of h, whose scale is 1),
    the tolerance, pass/fail, what was compared, and the oracle's seconds on this host
    (with the thread count).  The large GEMMs compare 256 rows x all columns; their full
    oracle time is extrapolated from that sample."""
    import torch
    import oracle
    from synth import workloads

    threads = oracle.max_threads()
    res = {}

    def nerr(out, ref, S):
        out = np.asarray(out, np.float64)
        if not np.all(np.isfinite(out)):
            return float("inf")
        m = S > 0
        e = float(np.max(np.abs(out - ref)[m] / S[m])) if np.any(m) else 0.0
        if np.any(~m) and not np.array_equal(out[~m], ref[~m]):
            e = float("inf")
        return e

    def record(name, err, tol, checked, t_oracle, scale=1.0):
        res[name] = {"max_norm_err": err, "tol": tol, "pass": bool(err <= tol), "checked": checked,
                     "oracle_s": round(t_oracle, 3), "cores": threads}
        if scale != 1.0:
            res[name]["oracle_full_s_extrapolated"] = round(t_oracle * scale, 1)

    def host(t):
        return t.detach().float().cpu().numpy().astype(np.float64)

    # fp32 GEMM 128^3
    d = workloads.gemm_small_fp32()
    C = isam.gemm(gpu(d["A"]), gpu(d["B"]))
    torch.cuda.synchronize()
    t = time.perf_counter()
    ref, S = oracle.gemm(d["A"], d["B"], 128, 128, 128)
    record("gemm_128x128x128_f32", nerr(host(C), ref, S), 1e-5, "all elements", time.perf_counter() - t)
    # skinny 4096 x 32 x 4096, bf16 and fp32
    d = workloads.skinny()
    for tag, A, B, tol in (("bf16", d["A_bf16"], d["B_bf16"], 1e-2), ("f32", d["A"], d["B"], 1e-5)):
        C = isam.gemm(gpu(A), gpu(B))
        torch.cuda.synchronize()
        t = time.perf_counter()
        ref, S = oracle.gemm(A, B, 4096, 32, 4096)
        record(f"skinny_4096x32x4096_{tag}", nerr(host(C), ref, S), tol, "all elements", time.perf_counter() - t)
    # GRU T64 B32 I=H=1024, bf16 weights
    d = workloads.gru()
    hs, _ = isam.gru_forward(gpu(d["x_bf16"]), gpu(d["W_bf16"]), gpu(d["U_bf16"]), bias=gpu(d["bias"]))
    torch.cuda.synchronize()
    t = time.perf_counter()
    ref = oracle.gru(d["x_bf16"], d["W_bf16"], d["U_bf16"], d["bias"], None, None)
    got = host(hs)
    err = float(np.max(np.abs(got - ref))) if np.all(np.isfinite(got)) else float("inf")
    record("gru_T64_B32_H1024_bf16", err, 1e-2, "every step of all 32 sequences (absolute error of h)",
           time.perf_counter() - t)
    # separable conv 32x56x56x128 -> 256
    d = workloads.dwsep()
    for tag, X, D, P, odt, tol in (("bf16_out_f32", d["X_bf16"], d["D_bf16"], d["P_bf16"], torch.float32, 1e-2),
                                   ("bf16_out_bf16", d["X_bf16"], d["D_bf16"], d["P_bf16"], torch.bfloat16, 1e-2),
                                   ("f32", d["X"], d["D"], d["P"], torch.float32, 1e-5)):
        y = isam.dwsep_conv(gpu(X), gpu(D), gpu(P), out_dtype=odt)
        torch.cuda.synchronize()
        t = time.perf_counter()
        Z, S = oracle.dwsep(X, D, P)
        record(f"dwsep_32x56x56x128_256_{tag}", nerr(host(y), Z, S), tol, "all elements", time.perf_counter() - t)
    del d
    # large bf16 GEMMs: 256 sampled rows (first and last included) x all columns
    for tag, d in (("8192x8192x8192", workloads.gemm_square_bf16()), ("8192x1024x16384", workloads.gemm_rect_bf16())):
        A_h, B_h = d["A_bf16"], d["B_bf16"]
        M, K = A_h.shape
        N = B_h.shape[1]
        rows = workloads.rows_sample(M, 256)
        Ag, Bg = gpu(A_h), gpu(B_h)
        t = time.perf_counter()
        ref, S = oracle.gemm(np.ascontiguousarray(A_h[rows]), B_h, len(rows), N, K)
        t_or = time.perf_counter() - t
        idx = torch.as_tensor(rows, device=Ag.device)
        for odt, otag in ((torch.bfloat16, "bf16"), (torch.float32, "f32")):
            C = isam.gemm(Ag, Bg, out_dtype=odt)
            torch.cuda.synchronize()
            record(f"gemm_{tag}_bf16_out_{otag}", nerr(host(C[idx]), ref, S), 1e-2,
                   f"{len(rows)} of {M} rows x all {N} columns", t_or, scale=M / len(rows))
            del C
        del Ag, Bg
    return res


def sources_hash(names) -> str:
    """sha256 over the named library sources under csrc/ (names and contents)."""
    import hashlib
    h = hashlib.sha256()
    for n in sorted(names):
        h.update(n.encode())
        with open(os.path.join(ROOT, "paper_1810_09958_amd", "csrc", n), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(name: str):
    """Traffic per launch recorded under profiles/, or None when any source the kernel is
    built from (the record lists them) changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", name)
    try:
        with open(path) as fh:
            rec = json.load(fh)
        if rec.get("sources_sha256") != sources_hash(rec["sources"]):
            return None
    except (OSError, ValueError, KeyError, TypeError):
        return None
    return rec.get("traffic_bytes_per_dispatch")


def cpu_baseline():
    """The CPU oracle (fp64, as used for parity) on a bounded sample of the square GEMM:
    R full rows of C = A.B with K = 8192, timed on this host's cores."""
    import oracle
    from synth import workloads

    sq = workloads.gemm_square_bf16()
    A, B = sq["A_bf16"], sq["B_bf16"]
    threads = oracle.max_threads()
    # pilot, then scale the sample to 10-15 s of oracle work (the pilot's fixed costs make it
    # overestimate the per-row time about twofold, hence the 24 s target)
    rows = max(32, 2 * threads)
    t = time.perf_counter()
    oracle.gemm(np.ascontiguousarray(A[:rows]), B, rows, 8192, 8192, with_norm=False)
    dt = time.perf_counter() - t
    rows2 = int(min(8192, rows * 24.0 / max(dt, 1e-3)))
    rows2 = max(threads, (rows2 // threads) * threads)
    t = time.perf_counter()
    oracle.gemm(np.ascontiguousarray(A[:rows2]), B, rows2, 8192, 8192, with_norm=False)
    dt2 = time.perf_counter() - t
    fl = 2.0 * rows2 * 8192 * 8192
    return {"value": round(fl / dt2 / 1e12, 6), "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"{rows2} rows of the 8192^3 bf16 GEMM (fp64 naive loops), {dt2:.1f} s"}


if __name__ == "__main__":
    main()
