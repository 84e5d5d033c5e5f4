#!/usr/bin/env python3
"""Benchmark of the EntQuant decode path on one MI355X.

Workload: the Llama-70B-shaped MLP pair, an 8192x28672 and a 28672x8192 BF16
matrix (Student-t(4) entries, log-normal(0, 0.5) row scales), quantised to
E4M3 at ~2.0 bits/param entropy and entropy-coded in 65536-symbol chunks.
One step runs the whole decode path on both matrices: decode to BF16, fused
decode-GEMV at batch 1 and fused decode-GEMV at batch 8 (6 launches).
Containers are resident in HBM before timing starts; several copies are
rotated so that compressed reads are not served from the 256 MB MALL.

Prints one JSON line: the decode throughput of the whole step, per-kernel
times (mean and p10/p50/p90), the HBM fraction of every kernel, the ALU
roofline of the dominant kernel and the oracle's CPU throughput.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published
# Vector ALU: 256 CUs x 4 SIMDs x 16 lanes, one 32-bit lane-op per lane and
# clock at 2.4 GHz (packed FP32 not counted: the path is integer work).
ALU_PEAK_TOPS = 256 * 64 * 2.4e9 / 1e12
# Algorithmic 32-bit lane-ops per decoded symbol: the decode step (slot
# mask, slot index, x >> P, multiply-add, renormalisation compare, two-part
# lane prefix count, word address, shift-or and select = 10) plus the use of
# the symbol: BF16 output 1 (row-table address); GEMV 1 (byte pick and
# conversion, per symbol pair) + B/2 (one dot2 per pair and batch row).
ALG_OPS = {"bf16": 11.0, "gemv1": 10.0 + 0.5 + 0.5 + 0.5, "gemv8": 10.0 + 0.5 + 0.5 + 4.0}
# Kernel (function) name of each op family's decode launch on these shapes.
KERNEL = {"bf16": "decode_kernel<4, 1, true, 0, 1>", "gemv1": "decode_kernel<4, 2, true, 1, 1>",
          "gemv8": "gemv_tiled_kernel<4, 8>"}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_config4.json")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2601_22787_amd", "csrc", "eq_decode.hip")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--copies", type=int, default=5,
                    help="container copies rotated across steps (defeats the MALL)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=8.0,
                    help="target CPU time of each oracle baseline sample (1 thread, all threads)")
    ap.add_argument("--cpu-threads", type=int, default=0,
                    help="oracle threads for the all-cores sample (0: host CPUs, at most 16)")
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


def cpu_baseline(layers, target_s, threads):
    """The oracle, as written, on a bounded sample: the first R rows of the
    8192x28672 matrix decoded from its container chunk by chunk, dequantised
    to BF16 and multiplied by one activation row in fp64.  Timed on one
    thread, then with `threads` threads over independent chunks and row
    blocks (the oracle's C routines release the interpreter lock)."""
    import numpy as np

    import oracle
    import synth
    spec, w, blob, _ = layers[0]
    info = oracle.container_info(blob)
    N, C = info.cols, info.chunk_syms
    scale = oracle.container_scales(blob)
    x = synth.activations(spec, 1)

    def run(R, T):
        t0 = time.perf_counter()
        nchunks = (R * N + C - 1) // C
        q = np.empty(nchunks * C, dtype=np.uint8)

        def dec(c):
            rc, qc = oracle.container_decode_chunk(blob, c)
            assert rc == oracle.OK
            q[c * C:c * C + qc.size] = qc

        def rows(r0, r1):
            w_hat = oracle.dequant(q[r0 * N:r1 * N].reshape(r1 - r0, N), scale[r0:r1])
            oracle.gemv(w_hat, x)

        if T == 1:
            for c in range(nchunks):
                dec(c)
            rows(0, R)
        else:
            with ThreadPoolExecutor(T) as ex:
                list(ex.map(dec, range(nchunks)))
                step = (R + T - 1) // T
                list(ex.map(lambda r0: rows(r0, min(R, r0 + step)), range(0, R, step)))
        return time.perf_counter() - t0

    def sample(T):
        R0 = 8 * T
        t0 = run(R0, T)
        R = int(min(info.rows, max(R0, R0 * target_s / max(t0, 1e-6))))
        return R, run(R, T)

    R1, t1 = sample(1)
    RT, tT = sample(threads)
    return {"value": RT * N / tT / 1e9, "unit": "Gparams/s", "cores": threads, "kind": "oracle",
            "sample": f"first {RT} rows ({RT * N} params) of the 8192x28672 matrix: oracle rANS "
                      f"decode per chunk + BF16 dequantisation + fp64 GEMV (B=1) on {threads} "
                      f"threads over chunks and row blocks, {tT:.1f}s",
            "single_thread_value": R1 * N / t1 / 1e9,
            "single_thread_sample": f"first {R1} rows, one thread, {t1:.1f}s"}


def traffic_per_launch(op):
    """HBM bytes of one launch of `op`'s decode kernel, from the committed
    FETCH_SIZE / WRITE_SIZE counter summary, scaled by the counters' readings
    for a copy of known size; None if that summary was taken on another
    version of the kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
        with open(KERNEL_SOURCE, "rb") as f:
            sha = hashlib.sha256(f.read()).hexdigest()
    except OSError:
        return None
    if t.get("source_sha256") != sha or op not in t.get("kernels", {}):
        return None
    return t["kernels"][op]["hbm_bytes"]


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
        q10, q50, q90 = (1000.0 * float(v) for v in np.percentile(ts, [10, 50, 90]))
        nbytes = algorithmic_bytes(infos[mi], op, B)
        comp = infos[mi]["file_bytes"] - 2 * (infos[mi]["padded_words"] - infos[mi]["total_words"])
        tops = ALG_OPS[op] * spec.params / us / 1e6
        kernels[f"{spec.name}.{op}"] = {
            "us": round(us, 2), "us_p10": round(q10, 2), "us_p50": round(q50, 2),
            "us_p90": round(q90, 2), "gparams_per_s": round(spec.params / us / 1e3, 1),
            "alg_bytes": nbytes, "gbs": round(nbytes / us / 1e3, 1),
            "hbm_frac": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4),
            "hbm_frac_compressed": round(comp / us / 1e3 / HBM_PEAK_GBS, 4),
            "alg_ops_per_param": ALG_OPS[op], "tops": round(tops, 2),
            "alu_frac": round(tops / ALU_PEAK_TOPS, 4)}
    # dominant kernel: the op family with the largest share of the step;
    # figures per launch (mean over the two matrices)
    fam = {}
    for (mi, op), ts in per.items():
        fam[op] = fam.get(op, 0.0) + sum(ts) / len(ts)
    dom = max(fam, key=fam.get)
    nmat = len(specs)
    dom_us = 1000.0 * fam[dom] / nmat
    dom_bytes = sum(algorithmic_bytes(infos[mi], dom, 8 if dom == "gemv8" else 1)
                    for mi in range(nmat)) / nmat
    dom_ops = ALG_OPS[dom] * sum(s.params for s in specs) / nmat
    achieved_gbs = dom_bytes / dom_us / 1e3
    achieved_tops = dom_ops / dom_us / 1e6

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
        "roofline": {"bound": "alu", "kernel": KERNEL[dom], "op": dom,
                     "achieved": round(achieved_tops, 2), "peak": round(ALU_PEAK_TOPS, 2),
                     "unit": "Tops/s", "frac": round(achieved_tops / ALU_PEAK_TOPS, 4),
                     "traffic": traffic_per_launch(dom),
                     "alg_bytes": round(dom_bytes), "us_per_launch": round(dom_us, 2),
                     "hbm": {"achieved": round(achieved_gbs, 1), "peak": HBM_PEAK_GBS,
                             "unit": "GB/s", "frac": round(achieved_gbs / HBM_PEAK_GBS, 4)}},
        "kernels": kernels,
        "copy_reference_gbs": round(copy_gbs, 1),
        "wall_s_timed": round(wall, 3),
    }
    if not args.no_cpu_baseline:
        threads = args.cpu_threads or min(16, os.cpu_count() or 1)
        result["cpu_baseline"] = cpu_baseline(layers, args.cpu_seconds, threads)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
