#!/usr/bin/env python3
"""Benchmark of the EntQuant decode path on one MI355X.

Workload: the Llama-70B-shaped MLP pair, an 8192x28672 and a 28672x8192 BF16
matrix (Student-t(4) entries, log-normal(0, 0.5) row scales), quantised to
E4M3 at ~2.0 bits/param entropy and entropy-coded in 65536-symbol chunks.
One step runs the whole decode path on both matrices: decode to BF16, fused
decode-GEMV at batch 1 and fused decode-GEMV at batch 8 (6 launches).
Containers are resident in HBM before timing starts; several copies are
rotated so that compressed reads are not served from the 256 MB MALL.

Prints one JSON line (see README of the bench contract in the design doc).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--copies", type=int, default=5,
                    help="container copies rotated across steps (defeats the MALL)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle baseline sample")
    return ap.parse_args()


def build_layers(eq, synth, specs, copies, dev):
    """Encode each matrix once (product encoder), upload `copies` copies."""
    out = []
    for spec in specs:
        t0 = time.time()
        w = synth.weights(spec)
        alpha, _ = eq.eqe_alpha_search(w, spec.target_bits, sample_rows=512)
        blob = eq.eqe_encode(w, alpha, chunk_syms=spec.chunk_syms, lanes=spec.lanes,
                             seed=spec.seed, target_bits=spec.target_bits)
        layers = [eq.Layer(blob, dev) for _ in range(copies)]
        print(f"[bench] {spec.name} {spec.rows}x{spec.cols}: container {blob.size / 1e6:.1f} MB "
              f"built in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)
        out.append((spec, w, blob, layers))
    return out


def blob_info(blob):
    """Header fields needed for byte accounting (read directly; no oracle)."""
    import numpy as np
    h = blob[:256]
    u32 = h.view(np.uint32)
    u64 = h.view(np.uint64)
    return dict(rows=int(u32[4]), cols=int(u32[5]), total_words=int(u64[6]),
                padded_words=int(u64[7]), entropy=float(h[80:84].view(np.float32)[0]),
                file_bytes=int(u64[17]))


def algorithmic_bytes(info, op, B):
    """Bytes one launch must move at minimum: the container (without its zero
    padding) in, plus the op's outputs/inputs."""
    n = info["rows"] * info["cols"]
    cont = info["file_bytes"] - 2 * (info["padded_words"] - info["total_words"])
    if op == "bf16":
        return cont + 2 * n
    return cont + 2 * B * info["cols"] + 4 * B * info["rows"]


def cpu_baseline(layers, target_s):
    """The oracle (single-threaded, as written) on a bounded sample: the first
    R rows of the 8192x28672 matrix, decoded from its container, dequantised to
    BF16 and multiplied by one activation row in fp64."""
    import numpy as np

    import oracle
    import synth
    spec, w, blob, _ = layers[0]
    info = oracle.container_info(blob)
    N, C = info.cols, info.chunk_syms
    scale = oracle.container_scales(blob)
    x = synth.activations(spec, 1)

    def run(R):
        t0 = time.perf_counter()
        nchunks = (R * N + C - 1) // C
        q = np.empty(nchunks * C, dtype=np.uint8)
        for c in range(nchunks):
            rc, qc = oracle.container_decode_chunk(blob, c)
            assert rc == oracle.OK
            q[c * C:c * C + qc.size] = qc
        q = q[:R * N].reshape(R, N)
        w_hat = oracle.dequant(q, scale[:R])
        oracle.gemv(w_hat, x)
        return time.perf_counter() - t0

    R0 = 16
    t0 = run(R0)
    R = int(min(info.rows, max(R0, R0 * target_s / max(t0, 1e-6))))
    t = run(R)
    return {"value": R * N / t / 1e9, "unit": "Gparams/s", "cores": 1, "kind": "oracle",
            "sample": f"first {R} rows ({R * N} params) of the 8192x28672 matrix: oracle "
                      f"rANS decode + BF16 dequantisation + fp64 GEMV (B=1), one thread, "
                      f"{t:.1f}s"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU; --gpus {args.gpus} is not supported "
              f"(the path would shard by output rows, see DESIGN.md)", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_2601_22787_amd as eq
    import synth
    from synth.configs import config_matrices

    eq.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    specs = config_matrices(4)
    layers = build_layers(eq, synth, specs, args.copies, dev)
    ops = ["bf16", "gemv1", "gemv8"]

    # device buffers shared by all steps
    nmax = max(s.params for s in specs)
    wout = torch.empty(nmax, dtype=torch.int16, device=dev)
    bufs = []
    for spec, w, blob, lays in layers:
        d = {}
        for B in (1, 8):
            x = torch.from_numpy(synth.activations(spec, B).view(np.int16)).to(dev)
            y = torch.empty(B, spec.rows, dtype=torch.float32, device=dev)
            d[B] = (x, y, lays[0].workspace(B))
        bufs.append(d)
    infos = [blob_info(blob) for _, _, blob, _ in layers]

    def launch(op, mi, L):
        if op == "bf16":
            eq.eq_decode_bf16(L, wout)
        else:
            B = 1 if op == "gemv1" else 8
            x, y, ws = bufs[mi][B]
            eq.eq_decode_gemv(L, x, B, None, y, ws)

    def one_step(s, timers=None):
        for mi, (spec, w, blob, lays) in enumerate(layers):
            L = lays[s % len(lays)]
            for op in ops:
                if timers is None:
                    launch(op, mi, L)
                else:
                    e0 = torch.cuda.Event(enable_timing=True)
                    e1 = torch.cuda.Event(enable_timing=True)
                    e0.record()
                    launch(op, mi, L)
                    e1.record()
                    timers.append((mi, op, e0, e1))

    # Reference: a plain device-to-device copy of 256 MiB, the known-size
    # kernel against which HBM byte counters are calibrated.
    ref_src = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
    ref_dst = torch.empty_like(ref_src)
    ref_dst.copy_(ref_src)
    c0 = torch.cuda.Event(enable_timing=True)
    c1 = torch.cuda.Event(enable_timing=True)
    c0.record()
    ref_dst.copy_(ref_src)
    c1.record()
    torch.cuda.synchronize()
    copy_gbs = 2 * ref_src.numel() / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del ref_src, ref_dst

    for s in range(args.warmup):
        one_step(s)
    torch.cuda.synchronize()
    for _, _, _, lays in layers:
        for L in lays:
            rc = eq.eq_get_status(L)
            if rc != eq.EQ_OK:
                raise RuntimeError(f"decode status {eq.eq_strerror(rc)}")

    timers = []
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record()
    for s in range(args.steps):
        one_step(args.warmup + s, timers)
    t_end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = t_start.elapsed_time(t_end)
    ms_per_step = total_ms / args.steps

    per = {}
    for mi, op, e0, e1 in timers:
        per.setdefault((mi, op), []).append(e0.elapsed_time(e1))
    kernels = {}
    for (mi, op), ts in per.items():
        spec = specs[mi]
        B = 8 if op == "gemv8" else 1
        us = 1000.0 * sum(ts) / len(ts)
        nbytes = algorithmic_bytes(infos[mi], op, B)
        comp = infos[mi]["file_bytes"] - 2 * (infos[mi]["padded_words"] - infos[mi]["total_words"])
        kernels[f"{spec.name}.{op}"] = {
            "us": round(us, 2), "gparams_per_s": round(spec.params / us / 1e3, 1),
            "alg_bytes": nbytes, "gbs": round(nbytes / us / 1e3, 1),
            "hbm_frac": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4),
            "hbm_frac_compressed": round(comp / us / 1e3 / HBM_PEAK_GBS, 4)}
    # dominant kernel: the op family with the largest share of the step
    fam = {}
    for (mi, op), ts in per.items():
        fam[op] = fam.get(op, 0.0) + sum(ts) / len(ts)
    dom = max(fam, key=fam.get)
    dom_bytes = sum(algorithmic_bytes(infos[mi], dom, 8 if dom == "gemv8" else 1)
                    for mi in range(len(specs)))
    dom_ms = fam[dom]
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9

    params_per_step = sum(s.params for s in specs) * len(ops)
    value = params_per_step / (ms_per_step * 1e-3) / 1e9

    result = {
        "metric": "decoded Gparams/s (decode->BF16 + fused decode-GEMV B=1,8 over the "
                  "8192x28672 and 28672x8192 layers); per-kernel us/layer and % HBM roofline",
        "value": round(value, 2), "unit": "Gparams/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u32", "data": "synthetic",
        "config": {"workload": "Llama-70B MLP layers 8192x28672 + 28672x8192, E4M3 at ~2.0 "
                               "bits/param, 65536-symbol chunks, 256 rANS lanes/chunk; per step "
                               "and matrix: " + ", ".join(ops),
                   "entropy_bits": [round(i["entropy"], 4) for i in infos],
                   "container_mb": [round(i["file_bytes"] / 1e6, 2) for i in infos],
                   "copies_rotated": args.copies},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None},
        "kernels": kernels,
        "copy_reference_gbs": round(copy_gbs, 1),
        "wall_s_timed": round(wall, 3),
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(layers, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
