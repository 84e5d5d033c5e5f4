#!/usr/bin/env python3
"""Benchmark of the EntQuant decode path on one MI355X.

Workload: the Llama-70B-shaped MLP pair, an 8192x28672 and a 28672x8192 BF16
matrix (Student-t(4) entries, log-normal(0, 0.5) row scales), quantised to
E4M3 at ~2.0 bits/param entropy and entropy-coded in 65536-symbol chunks.
One step runs the whole decode path on both matrices: decode to BF16, fused
decode-GEMV at batch 1 and fused decode-GEMV at batch 8 (5 launches), on
containers of version 1.  Containers are resident in HBM before timing
starts; every read of a matrix takes the next of several device copies, so
that no launch finds its compressed bytes in the 256 MB MALL.

Prints one JSON line: the decode throughput of the whole step, per-launch
times (GPU time from graph replay, and eager per-call events with
p10/p50/p90) and HBM fractions, the HBM roofline of the
dominant kernel, the target row (fused decode-GEMV at batch 1 on the
8192x28672 matrix, compressed bytes over time against the HBM peak) on both
container versions, every op on container version 2 (256 x 256 tiles of the
same codes), and the oracle's CPU throughput.
--base-format int8 runs the same workload coded with the Int8 base format
(the paper's alternative to Float8) instead of E4M3.  --workload selects
configs 1-3, the 80-layer stack or prefill instead.
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
# Kernel (function) name of each op family's decode launch on these shapes,
# container version 1 (template arguments: lanes / 64, op, [whole-row
# steps,] activation source, batch, base format).
KERNEL = {"bf16": "multi_decode_kernel<4, 1, 0, 1, 1>",
          "gemv1": "decode_kernel<4, 2, true, 1, 1, 1>", "gemv8": "gemv_tiled_kernel<4, 8, 1>"}
KERNEL_INT8 = {"bf16": "multi_decode_kernel<4, 1, 0, 1, 2>",
               "gemv1": "decode_kernel<4, 2, true, 1, 1, 2>", "gemv8": "gemv_tiled_kernel<4, 8, 2>"}
FORMATS = {"e4m3": 1, "int8": 2}
COUNTERS_FILE = os.path.join(ROOT, "profiles", "counters_config4.json")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2601_22787_amd", "csrc", f)
                  for f in ("eq_decode.hip", "eq_decode2.hip", "eq_device.h")]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--copies", type=int, default=5,
                    help="container copies rotated across steps (defeats the MALL)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--eager", action="store_true",
                    help="launch each timed step's kernels one by one instead of replaying a "
                         "captured HIP graph of the step")
    ap.add_argument("--cpu-seconds", type=float, default=8.0,
                    help="target CPU time of each oracle baseline sample (1 thread, all threads)")
    ap.add_argument("--workload", choices=("c4", "c5", "c123", "prefill"), default="c4",
                    help="c4: the 8192x28672 / 28672x8192 pair (default); c5: the 80-layer stack, "
                         "block-wise vs per-matrix, decode-GEMV B=1 and decode to BF16; c123: "
                         "every matrix of configs 1-3, decode to BF16 and decode-GEMV B=1; "
                         "prefill: the c4 pair at --tokens tokens, decode to codes + MFMA GEMM")
    ap.add_argument("--tokens", type=int, default=2048, help="prefill batch (tokens)")
    ap.add_argument("--container", type=int, choices=(1, 2), default=1,
                    help="c5 workload: container version of the stack's layers")
    ap.add_argument("--v2-tile-rows", type=int, choices=(64, 128, 256), default=0,
                    help="version-2 tile rows for every matrix (columns as v2_tiles sets them) "
                         "instead of the rule of v2_tiles")
    ap.add_argument("--row-order", action="store_true",
                    help="version-2 containers with the row order: tiles cut over the rows "
                         "sorted by their phrase count")
    ap.add_argument("--cpu-threads", type=int, default=0,
                    help="oracle threads for the all-cores sample (0: host CPUs, at most 16)")
    ap.add_argument("--base-format", choices=tuple(FORMATS), default="e4m3",
                    help="base format of the codes (c4 workload): E4M3 (default) or Int8")
    ap.add_argument("--counters-from", nargs="+", metavar="DIR",
                    help="no benchmark: summarise rocprofv3 --pmc output directories (FETCH_SIZE; "
                         "WRITE_SIZE + SQ_INSTS_VALU) of a run of this script into the counter "
                         "file the HBM traffic and VALU figures are read from")
    return ap.parse_args()


def v2_tiles(spec, rows=0):
    """Tile rows and columns of the version-2 containers.  The width sets the
    state bytes per code (32 bits per row segment), so it follows the chunk
    size: 256 columns for 65536-symbol chunks, C / 128 below.  The height is
    the taller of (256, 128), or of (128, 64) below 65536 symbols, when the
    matrix has at least 2048 such tiles (8 per compute unit), else the
    shorter: half the tile, the same bytes, twice the tiles and half the
    work per step, which shortens launches that cannot fill the GPU
    (batch-1 GEMV: config-5 attention matrices 43.5 -> 34 us, config 2
    19.8 -> 17.6 us, config 1 12.7 -> 9.2 us).  rows > 0 sets the height."""
    tall, tc = (256, 256) if spec.chunk_syms >= 65536 else (128, spec.chunk_syms // 128)
    if rows:
        return rows, tc
    tiles = -(-spec.rows // tall) * -(-spec.cols // tc)
    return (tall if tiles >= 2048 else tall // 2), tc


def build_layers(eq, synth, specs, copies, dev, fmt=1, v2_copies=0, row_order=False,
                 v2_rows=0):
    """Encode each matrix (product encoder) and upload `copies` device copies;
    with v2_copies > 0 also the same codes (same alpha) in container version
    2, tiles of v2_tiles(spec, v2_rows), with the row order if row_order."""
    out = []
    for spec in specs:
        t0 = time.time()
        w = synth.weights(spec)
        alpha, _ = eq.eqe_alpha_search(w, spec.target_bits, sample_rows=512, base_format=fmt)
        blob = eq.eqe_encode(w, alpha, chunk_syms=spec.chunk_syms, lanes=spec.lanes,
                             seed=spec.seed, target_bits=spec.target_bits, base_format=fmt)
        layers = [eq.Layer(blob, dev) for _ in range(copies)]
        item = {"spec": spec, "w": w, "blob": blob, "layers": layers}
        msg = f"container {blob.size / 1e6:.1f} MB"
        if v2_copies:
            tr, tc = v2_tiles(spec, v2_rows)
            blob2 = eq.eqe_encode2(w, alpha, tile_rows=tr, tile_cols=tc,
                                   seed=spec.seed, target_bits=spec.target_bits,
                                   base_format=fmt, row_order=row_order)
            item["blob2"] = blob2
            item["layers2"] = [eq.Layer(blob2, dev) for _ in range(v2_copies)]
            msg += f", version 2 {blob2.size / 1e6:.1f} MB"
        print(f"[bench] {spec.name} {spec.rows}x{spec.cols}: {msg} built in "
              f"{time.time() - t0:.1f}s", file=sys.stderr, flush=True)
        out.append(item)
    return out


def blob_info(blob):
    """Header fields needed for byte accounting (read directly; no oracle)."""
    import numpy as np
    h = blob[:256]
    u32 = h.view(np.uint32)
    u64 = h.view(np.uint64)
    return dict(rows=int(u32[4]), cols=int(u32[5]), total_words=int(u64[6]),
                padded_words=int(u64[7]), entropy=float(h[80:84].view(np.float32)[0]),
                file_bytes=int(u64[17]), lanes=int(u32[8]),
                tile_cols=int(u32[21]) if int(u32[1]) == 2 else 0)


def algorithmic_bytes(info, op, B):
    """Bytes one launch must move at minimum: the container (without its zero
    padding) in, plus the op's outputs/inputs."""
    n = info["rows"] * info["cols"]
    cont = info["file_bytes"] - 2 * (info["padded_words"] - info["total_words"])
    if op == "bf16":
        return cont + 2 * n
    return cont + 2 * B * info["cols"] + 4 * B * info["rows"]


def cpu_baseline(layers, target_s, threads, fmt=1):
    """The oracle, as written, on bounded samples, on `threads` host threads
    over independent chunks and row blocks (its C routines release the
    interpreter lock), median of three runs:
    - value: the first R rows of the 8192x28672 matrix decoded from its
      container chunk by chunk, dequantised to BF16 and multiplied by one
      activation row in fp64 (decode-GEMV, B = 1); also on one thread;
    - bf16: the same rows decoded and dequantised (decode to BF16);
    - config 5: one 1024x8192 row block per entropy class (2, 3, 4 bits,
      65536-symbol chunks) decoded, dequantised and multiplied; the seconds
      of an 80-layer pass extrapolated from the per-parameter times."""
    import numpy as np

    import oracle
    import paper_2601_22787_amd as eq
    import synth
    from synth.configs import MatrixSpec, STUDENT_T, matrix_seed

    def timer(blob, spec, gemv):
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
                w_hat = oracle.dequant(q[r0 * N:r1 * N].reshape(r1 - r0, N), scale[r0:r1], fmt)
                if gemv:
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

        def sample(T, seconds):
            # rows sized from a short probe run; then the median of three runs
            R0 = 8 * T
            t0 = run(R0, T)
            R = int(min(info.rows, max(R0, R0 * seconds / max(t0, 1e-6))))
            return R, N, sorted(run(R, T) for _ in range(3))[1]
        return sample

    spec, blob = layers[0]["spec"], layers[0]["blob"]
    R1, N, t1 = timer(blob, spec, True)(1, target_s)
    RT, _, tT = timer(blob, spec, True)(threads, target_s)
    RB, _, tB = timer(blob, spec, False)(threads, target_s / 2)
    # config 5, one row block per entropy class
    per_param = {}
    for cls, bits in enumerate((2.0, 3.0, 4.0)):
        sp = MatrixSpec(f"c5.class{cls}", 1024, 8192, STUDENT_T, 5, 0.5, 0.0, 0.0, bits, 65536,
                        256, matrix_seed(5, cls, 4))
        w = synth.weights(sp)
        alpha, _ = eq.eqe_alpha_search(w, bits, sample_rows=256, base_format=fmt)
        b5 = eq.eqe_encode(w, alpha, chunk_syms=65536, lanes=256, seed=sp.seed, target_bits=bits,
                           base_format=fmt)
        R5, N5, t5 = timer(b5, sp, True)(threads, target_s / 4)
        per_param[bits] = t5 / (R5 * N5)
    stack = {"q": (8192, 8192), "k": (1024, 8192), "v": (1024, 8192), "o": (8192, 8192),
             "gate": (28672, 8192), "up": (28672, 8192), "down": (8192, 28672)}
    layer_params = sum(m * n for m, n in stack.values())
    c5_seconds = sum(layer_params * per_param[(2.0, 3.0, 4.0)[l % 3]] for l in range(80))
    return {"value": RT * N / tT / 1e9, "unit": "Gparams/s", "cores": threads, "kind": "oracle",
            "sample": f"first {RT} rows ({RT * N} params) of the 8192x28672 matrix: oracle rANS "
                      f"decode per chunk + BF16 dequantisation + fp64 GEMV (B=1) on {threads} "
                      f"threads over chunks and row blocks, median of 3 runs, {tT:.1f}s each",
            "single_thread_value": R1 * N / t1 / 1e9,
            "single_thread_sample": f"first {R1} rows, one thread, median of 3 runs, {t1:.1f}s each",
            "bf16_value": RB * N / tB / 1e9,
            "bf16_sample": f"first {RB} rows of the 8192x28672 matrix: oracle decode + BF16 "
                           f"dequantisation (no GEMV) on {threads} threads, median of 3 runs, "
                           f"{tB:.1f}s each",
            "config5_seconds_per_pass": round(c5_seconds, 2),
            "config5_sample": "extrapolated: one 1024x8192 row block per entropy class (2, 3, 4 "
                              "bits) timed (oracle decode + dequantisation + fp64 GEMV B=1, "
                              f"{threads} threads); seconds per parameter of each class times "
                              "the parameters of the 80 layers (layer l in class l mod 3)"}


def kernel_counters(kernel):
    """HBM bytes (FETCH_SIZE + WRITE_SIZE, each scaled by the counters'
    readings for a copy of known size) and SQ_INSTS_VALU of one launch of
    `kernel`, from the committed counter summary; None if that summary was
    taken on other kernel sources."""
    try:
        with open(COUNTERS_FILE) as f:
            t = json.load(f)
    except OSError:
        return None
    if t.get("source_sha256") != kernel_source_sha():
        return None
    return t.get("kernels", {}).get(kernel)


def short_kernel_name(full):
    """'void (anonymous namespace)::decode_kernel<4, 2, true, 1, 1, 1>(...)'
    -> 'decode_kernel<4, 2, true, 1, 1, 1>'."""
    s = full.replace("(anonymous namespace)::", "").strip()
    if s.startswith("void "):
        s = s[5:]
    s = s.split("(")[0].strip()
    base, _, targs = s.partition("<")
    return base.split("::")[-1] + ("<" + targs if targs else "")


def summarise_counters(dirs):
    """Per-dispatch means of FETCH_SIZE, WRITE_SIZE (KiB) and SQ_INSTS_VALU per
    kernel over rocprofv3 counter-collection CSVs; HBM bytes scaled by the
    readings for the bench's 256 MiB device-to-device copy (read and written
    once: 2^28 bytes each way)."""
    import csv
    import glob
    import statistics
    vals, full = {}, {}
    for d in dirs:
        for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            with open(path) as f:
                for r in csv.DictReader(f):
                    short = short_kernel_name(r["Kernel_Name"])
                    full[short] = r["Kernel_Name"]
                    key = (short, r["Counter_Name"])
                    vals.setdefault(key, {}).setdefault(r["Dispatch_Id"], 0.0)
                    vals[key][r["Dispatch_Id"]] += float(r["Counter_Value"])
    per = {}
    for (k, c), d in vals.items():
        per.setdefault(k, {})[c] = (statistics.mean(d.values()), len(d))
    # the copy: torch's elementwise copy kernel, 256 MiB each way
    copies = [(abs(v["FETCH_SIZE"][0] - 262144.0), k) for k, v in per.items()
              if "FETCH_SIZE" in v and "WRITE_SIZE" in v and "copy_kernel" in full[k]]
    ref = min(copies)[1]
    f_fetch = 262144.0 / per[ref]["FETCH_SIZE"][0]
    f_write = 262144.0 / per[ref]["WRITE_SIZE"][0]
    out = {"source_sha256": kernel_source_sha(), "copy_kernel": ref,
           "copy_fetch_kib": round(per[ref]["FETCH_SIZE"][0], 1),
           "copy_write_kib": round(per[ref]["WRITE_SIZE"][0], 1),
           "scale_fetch": round(f_fetch, 5), "scale_write": round(f_write, 5), "kernels": {}}
    for k, v in sorted(per.items()):
        if "FETCH_SIZE" not in v or "WRITE_SIZE" not in v:
            continue
        e = {"fetch_kib": round(v["FETCH_SIZE"][0], 1), "write_kib": round(v["WRITE_SIZE"][0], 1),
             "dispatches": v["FETCH_SIZE"][1],
             "hbm_bytes": round(1024.0 * (f_fetch * v["FETCH_SIZE"][0] +
                                          f_write * v["WRITE_SIZE"][0]))}
        if "SQ_INSTS_VALU" in v:
            e["valu_insts"] = round(v["SQ_INSTS_VALU"][0])
        out["kernels"][k] = e
    with open(COUNTERS_FILE, "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)
    print(json.dumps(out, indent=1, sort_keys=True))


def kernel_source_sha():
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def run_env():
    """Device, software and host facts recorded with every result."""
    import platform
    import torch
    props = torch.cuda.get_device_properties(0)
    cpu = platform.processor() or ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    env = {"device": props.name, "arch": getattr(props, "gcnArchName", ""),
           "compute_units": props.multi_processor_count,
           "hbm_gib": round(props.total_memory / 2**30, 1), "hip": torch.version.hip,
           "torch": torch.__version__, "cpu": cpu, "host_cores": os.cpu_count()}
    env.update(gpu_clocks())
    return env


def gpu_clocks():
    """Shader and memory clock levels the driver lists in sysfs (MHz), with the
    level current when read; empty where the files are not readable."""
    import glob
    out = {}
    for kind, key in (("sclk", "sclk_mhz"), ("mclk", "mclk_mhz")):
        for path in sorted(glob.glob(f"/sys/class/drm/card*/device/pp_dpm_{kind}")):
            try:
                with open(path) as f:
                    levels = [ln.split(":", 1)[1].strip() for ln in f if ":" in ln]
            except OSError:
                continue
            if levels:
                out[key] = levels  # a trailing '*' marks the current level
                break
    return out


def run_stack(args):
    """Config 5: an 80-layer 70B-shaped stack (q/k/v/o 8192x8192, 1024x8192 x2,
    8192x8192; gate/up 28672x8192; down 8192x28672), layer l coded at
    (2, 3, 4)[l mod 3] bits.  One layer per entropy class is generated and
    encoded; the 80 layers are distinct device copies of those three (the
    kernels' work depends on the symbol statistics, not on the values, and
    every copy is read from HBM).  Timed per pass over all 80 layers:
    decode-GEMV at B = 1 block-wise (q|k|v and gate|up share their inputs;
    4 launches per layer) and per matrix (7 launches), and decode to BF16
    block-wise (one launch per layer into a block buffer) and per matrix."""
    import numpy as np
    import torch

    import paper_2601_22787_amd as eq
    import synth
    from synth.configs import config_matrices

    eq.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    names = ("q", "k", "v", "o", "gate", "up", "down")
    proto = []  # per entropy class: {name: (spec, blob)}
    for layer in range(3):
        t0 = time.time()
        d = {}
        for spec in config_matrices(5, layers=[layer]):
            w = synth.weights(spec)
            alpha, _ = eq.eqe_alpha_search(w, spec.target_bits, sample_rows=512)
            if args.container == 2:
                tr, tc = v2_tiles(spec, args.v2_tile_rows)
                blob = eq.eqe_encode2(w, alpha, tile_rows=tr, tile_cols=tc,
                                      seed=spec.seed, target_bits=spec.target_bits,
                                      row_order=args.row_order)
            else:
                blob = eq.eqe_encode(w, alpha, chunk_syms=spec.chunk_syms, lanes=spec.lanes,
                                     seed=spec.seed, target_bits=spec.target_bits)
            d[spec.name.split(".")[-1]] = (spec, blob)
        proto.append(d)
        mb = sum(b.size for _, b in d.values()) / 1e6
        print(f"[bench] stack class {layer}: {mb:.0f} MB in {time.time() - t0:.1f}s",
              file=sys.stderr, flush=True)
    nl = 80
    layers = [{n: eq.Layer(proto[l % 3][n][1], dev) for n in names} for l in range(nl)]
    params = sum(proto[l % 3][n][0].params for l in range(nl) for n in names)
    cont_bytes = sum(proto[l % 3][n][1].size for l in range(nl) for n in names)
    print(f"[bench] {nl} layers resident: {cont_bytes / 1e9:.2f} GB", file=sys.stderr, flush=True)
    # inputs of a block: attention input (q, k, v), o input, MLP input (gate, up), down input
    xs = {k: torch.from_numpy(synth.vector(0x5EED, 16 + i, n).view(np.int16)).to(dev).view(1, n)
          for i, (k, n) in enumerate((("attn", 8192), ("o", 8192), ("mlp", 8192), ("down", 28672)))}
    groups = ((("q", "k", "v"), "attn"), (("o",), "o"), (("gate", "up"), "mlp"), (("down",), "down"))
    ys = {n: torch.empty(1, proto[0][n][0].rows, dtype=torch.float32, device=dev) for n in names}
    ws_multi = {g: eq.multi_workspace([layers[0][n] for n in g], 1) for g, _ in groups}
    ws_one = {n: layers[0][n].workspace(1) for n in names}
    block_elems = sum(proto[0][n][0].params for n in names)
    wbuf = torch.empty(block_elems, dtype=torch.int16, device=dev)
    offs, o = {}, 0
    for n in names:
        offs[n] = o
        o += proto[0][n][0].params
    outs = [wbuf[offs[n]:offs[n] + proto[0][n][0].params] for n in names]

    def gemv_block(Lset):
        for g, xk in groups:
            eq.eq_decode_gemv_multi([Lset[n] for n in g], xs[xk], 1, None, [ys[n] for n in g],
                                    ws_multi[g])

    def gemv_matrix(Lset):
        for g, xk in groups:
            for n in g:
                eq.eq_decode_gemv(Lset[n], xs[xk], 1, None, ys[n], ws_one[n])

    def bf16_block(Lset):
        eq.eq_decode_bf16_multi([Lset[n] for n in names], outs)

    def bf16_matrix(Lset):
        for n, out in zip(names, outs):
            eq.eq_decode_bf16(Lset[n], out)

    def time_pass(fn, reps):
        for Lset in layers[:3]:
            fn(Lset)
        torch.cuda.synchronize()
        graph = None
        if not args.eager:  # the whole 80-layer pass as one HIP graph
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                for Lset in layers:
                    fn(Lset)
            graph.replay()
            torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            if graph is not None:
                graph.replay()
            else:
                for Lset in layers:
                    fn(Lset)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    res = {}
    for name, fn in (("gemv_b1_block", gemv_block), ("gemv_b1_per_matrix", gemv_matrix),
                     ("bf16_block", bf16_block), ("bf16_per_matrix", bf16_matrix)):
        ms = time_pass(fn, args.steps)
        res[name] = {"ms_per_pass": round(ms, 3), "us_per_layer": round(1000 * ms / nl, 1),
                     "gparams_per_s": round(params / ms / 1e6, 1)}
        print(f"[bench] {name}: {ms:.2f} ms per pass", file=sys.stderr, flush=True)
    for Lset in layers:
        for n in names:
            if eq.eq_get_status(Lset[n]) != eq.EQ_OK:
                raise RuntimeError("decode status not OK")
    gb = res["gemv_b1_block"]
    print(json.dumps({
        "metric": "decoded Gparams/s, 80-layer stack, fused decode-GEMV B=1 (block-wise launches)",
        "value": gb["gparams_per_s"], "unit": "Gparams/s", "n_gpus": 1, "steps": args.steps,
        "ms_per_step": gb["ms_per_pass"], "higher_is_better": True, "vs_baseline": None,
        "dtype": "u32", "data": "synthetic", "env": run_env(),
        "config": {"workload": "config 5: 80 layers x {q 8192x8192, k/v 1024x8192, o 8192x8192, "
                               "gate/up 28672x8192, down 8192x28672}, (2,3,4)[l mod 3] bits, "
                               "65536-symbol chunks (version 2: tiles of 256 columns, 128 rows "
                               "for q/k/v/o, 256 for gate/up/down); 3 distinct layers, 80 device "
                               "copies",
                   "container": args.container,
                   "v2_row_order": bool(args.row_order and args.container == 2),
                   "launch": "eager" if args.eager else "HIP graph of each 80-layer pass",
                   "params": params, "container_gb": round(cont_bytes / 1e9, 3),
                   "hbm_frac_compressed_block_gemv": round(
                       cont_bytes / (gb["ms_per_pass"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
        "passes": res}), flush=True)


def run_small(args):
    """Configs 1-3 (1024x1024; the 4096x4096 Llama-2-7B attention projection;
    its 11008x4096 / 4096x11008 MLP matrices): for each matrix, decode to BF16
    and the fused decode-GEMV at B = 1 and 8, each launch timed alone with HIP events
    over `--copies` rotated container copies.  Reports us per launch,
    Gparams/s and the fraction of the HBM peak on the algorithmic bytes."""
    import numpy as np
    import torch

    import paper_2601_22787_amd as eq
    import synth
    from synth.configs import config_matrices

    eq.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    rows = []

    def time_op(fn, lays):
        for i in range(args.warmup):
            fn(lays[i % len(lays)])
        ev = []
        for i in range(args.steps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            fn(lays[i % len(lays)])
            e1.record()
            ev.append((e0, e1))
        torch.cuda.synchronize()
        return [1000.0 * a.elapsed_time(b) for a, b in ev]

    for cfg in (1, 2, 3):
        specs = config_matrices(cfg)
        for item in build_layers(eq, synth, specs, args.copies, dev, v2_copies=args.copies,
                                 row_order=args.row_order, v2_rows=args.v2_tile_rows):
            spec = item["spec"]
            out = torch.empty(spec.params, dtype=torch.int16, device=dev)
            x = torch.from_numpy(synth.activations(spec, 1).view(np.int16)).to(dev)
            y = torch.empty(1, spec.rows, dtype=torch.float32, device=dev)
            x8 = torch.from_numpy(synth.activations(spec, 8).view(np.int16)).to(dev)
            y8 = torch.empty(8, spec.rows, dtype=torch.float32, device=dev)
            for version, blob, lays in ((1, item["blob"], item["layers"]),
                                        (2, item["blob2"], item["layers2"])):
                info = blob_info(blob)
                ws = lays[0].workspace(8)
                fns = {"bf16": lambda L: eq.eq_decode_bf16(L, out),
                       "gemv1": lambda L, ws=ws: eq.eq_decode_gemv(L, x, 1, None, y, ws),
                       "gemv8": lambda L, ws=ws: eq.eq_decode_gemv(L, x8, 8, None, y8, ws)}
                for op, fn in fns.items():
                    ts = time_op(fn, lays)
                    us_eager = sum(ts) / len(ts)
                    us = us_eager if args.eager else time_graph(
                        lambda i, fn=fn: fn(lays[i]), len(lays), 3)
                    nbytes = algorithmic_bytes(info, op, 8 if op == "gemv8" else 1)
                    rows.append({"config": cfg, "matrix": spec.name,
                                 "shape": [spec.rows, spec.cols], "container": version,
                                 "tile": ([info["lanes"], info["tile_cols"]] if version == 2
                                          else None),
                                 "chunk_syms": spec.chunk_syms, "lanes": spec.lanes,
                                 "entropy_bits": round(info["entropy"], 4),
                                 "container_mb": round(info["file_bytes"] / 1e6, 3), "op": op,
                                 "us": round(us, 2), "us_eager": round(us_eager, 2),
                                 "us_eager_p50": round(float(np.percentile(ts, 50)), 2),
                                 "gparams_per_s": round(spec.params / us / 1e3, 1),
                                 "hbm_frac": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4)})
                    print(f"[bench] config {cfg} {spec.name} v{version} {op}: {us:.1f} us",
                          file=sys.stderr, flush=True)
                for L in lays:
                    if eq.eq_get_status(L) != eq.EQ_OK:
                        raise RuntimeError("decode status not OK")
            del item, out
            torch.cuda.empty_cache()
    # headline: the faster container per matrix for the batch-1 GEMV
    best = {}
    for r in rows:
        if r["op"] == "gemv1":
            k = (r["config"], r["matrix"])
            if k not in best or r["us"] < best[k]["us"]:
                best[k] = r
    params = sum(r["shape"][0] * r["shape"][1] for r in best.values())
    us_gemv = sum(r["us"] for r in best.values())
    print(json.dumps({
        "metric": "decoded Gparams/s, configs 1-3, fused decode-GEMV B=1 over every matrix "
                  "(launches timed one by one; the faster container version per matrix)",
        "value": round(params / us_gemv / 1e3, 1), "unit": "Gparams/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "higher_is_better": True,
        "vs_baseline": None, "dtype": "u32", "data": "synthetic",
        "config": {"workload": "config 1: 1024x1024, 2 bits, 4096-symbol chunks; config 2: "
                               "4096x4096, 3 bits, 16384-symbol chunks; config 3: 11008x4096 x2 "
                               "and 4096x11008 with 0.1% outliers, 2 bits, 16384-symbol chunks",
                   "v2_row_order": bool(args.row_order),
                   "copies_rotated": args.copies},
        "matrices": rows, "env": run_env()}), flush=True)


MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix throughput, published


def run_prefill(args):
    """Prefill of the config-4 pair: per matrix, the codes decoded into the
    workspace and the W8A16 MFMA GEMM over --tokens tokens (eq_decode_gemm).
    Roofline of the GEMM kernel: 2 M N B flops per launch against the dense
    bf16 peak."""
    import numpy as np
    import torch

    import paper_2601_22787_amd as eq
    import synth
    from synth.configs import config_matrices

    eq.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    fmt = FORMATS[args.base_format]
    specs = config_matrices(4)
    layers = build_layers(eq, synth, specs, 1, dev, fmt)
    B = args.tokens
    bufs = []
    for item in layers:
        spec, lays = item["spec"], item["layers"]
        x = torch.from_numpy(np.stack([synth.vector(spec.seed, 100 + t % 64, spec.cols)
                                       for t in range(B)]).view(np.int16)).to(dev)
        y = torch.empty(B, spec.rows, dtype=torch.float32, device=dev)
        bufs.append((lays[0], x, y, lays[0].gemm_workspace(B)))

    def step(timers=None):
        for mi, (L, x, y, ws) in enumerate(bufs):
            code_bytes = (L.rows * L.cols + 255) // 256 * 256
            codes, part = ws[:L.rows * L.cols], ws[code_bytes:]
            part = part if part.numel() else None
            for op, fn in (("decode_codes", lambda: eq.eq_decode_codes(L, codes)),
                           ("gemm", lambda: eq.eq_gemm_codes(L, codes, x, B, None, y, part))):
                if timers is None:
                    fn()
                    continue
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
                fn()
                e1.record()
                timers.append((mi, op, e0, e1))

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    timers = []
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(args.steps):
        step(timers)
    t1.record()
    torch.cuda.synchronize()
    for L, _, _, _ in bufs:
        if eq.eq_get_status(L) != eq.EQ_OK:
            raise RuntimeError("decode status not OK")
    ms = t0.elapsed_time(t1) / args.steps
    per = {}
    for mi, op, e0, e1 in timers:
        per.setdefault((mi, op), []).append(e0.elapsed_time(e1) * 1000.0)
    kernels, g_us, g_flops = {}, 0.0, 0.0
    for (mi, op), ts in sorted(per.items()):
        spec = specs[mi]
        us = float(np.mean(ts))
        d = {"us": round(us, 2), "us_p50": round(float(np.median(ts)), 2)}
        if op == "gemm":
            flops = 2.0 * spec.params * B
            d["tflops"] = round(flops / us / 1e6, 1)
            d["mfma_frac"] = round(flops / us / 1e6 / MFMA_BF16_PEAK_TFLOPS, 4)
            g_us += us
            g_flops += flops
        else:
            d["gparams_per_s"] = round(spec.params / us / 1e3, 1)
        kernels[f"{spec.name}.{op}"] = d
    achieved = g_flops / g_us / 1e6
    params = sum(s.params for s in specs)
    print(json.dumps({
        "metric": "prefill tokens/s through the 8192x28672 and 28672x8192 layers (decode to codes "
                  "+ W8A16 MFMA GEMM); GEMM TFLOP/s and % of the bf16 matrix peak",
        "value": round(B / (ms * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "env": run_env(),
        "config": {"workload": f"prefill of the Llama-70B MLP pair 8192x28672 + 28672x8192, "
                               f"{args.base_format.upper()} codes at ~2.0 bits/param, {B} tokens",
                   "tokens": B, "params": params, "base_format": args.base_format},
        "roofline": {"bound": "mfma", "kernel": "gemm_codes_kernel", "op": "gemm",
                     "achieved": round(achieved, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4),
                     "traffic": None, "us_per_launch": round(g_us / len(specs), 2)},
        "kernels": kernels}), flush=True)


# (template arguments: tile rows / 64, op, batch, packed table entries)
V2_KERNEL = {"gemv1": "decode2_kernel<4, 2, 1, false, false>",
             "gemv8": "decode2_kernel<4, 2, 8, false, false>",
             "bf16": "decode2_kernel<4, 1, 1, true, false>",
             "codes": "decode2_kernel<4, 0, 1, true, false>"}
TARGET_FRAC = 0.60  # fused decode-GEMV B=1 on 8192x28672, compressed bytes / HBM peak


def time_eager(fn, n, reps):
    """Mean, p50 and all per-launch times (us) of fn(i) for i < reps, each
    bracketed by HIP events on the current stream (the library's stream)."""
    import numpy as np
    import torch
    ev = []
    for i in range(reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        fn(i)
        e1.record()
        ev.append((e0, e1))
    torch.cuda.synchronize()
    ts = [1000.0 * e0.elapsed_time(e1) for e0, e1 in ev]
    return float(np.mean(ts)), float(np.median(ts)), ts


def time_graph(fn, calls, reps):
    """Mean time (us) per call of fn(0) .. fn(calls - 1), captured back to back
    in one HIP graph (the sequence repeated to about 40 calls, so that the
    gap between two replays is spread thin) and replayed reps times between
    two HIP events: the GPU time of the calls' kernels without the host's
    launch and event gaps.  Replays for at least 20 ms first (at least two),
    so that the timed ones run at the GPU's working clocks."""
    import torch
    rounds = max(1, -(-40 // calls))
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(rounds):
            for i in range(calls):
                fn(i)
    t0 = time.time()
    for k in range(1000):
        g.replay()
        torch.cuda.synchronize()
        if k >= 1 and time.time() - t0 >= 0.02:
            break
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return 1000.0 * e0.elapsed_time(e1) / (reps * rounds * calls)


def hbm_reference(torch, dev):
    """Achievable HBM bandwidth on this device: a 1 GiB same-type device copy
    (bytes read + written) and a 1 GiB streaming read (a sum over float32),
    each the best of 5 runs timed with HIP events.  The roofline's
    denominator stays the published 8 TB/s."""
    n = 1 << 28  # 1 GiB of 4-byte words
    src = torch.zeros(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    out = {}
    for name, fn, nbytes in (("copy_gbs", lambda: dst.copy_(src), 2 * 4 * n),
                             ("read_gbs", lambda: torch.sum(src), 4 * n)):
        fn()
        best = float("inf")
        for _ in range(5):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            best = min(best, e0.elapsed_time(e1) * 1e-3)
        out[name] = round(nbytes / best / 1e9, 1)
    del src, dst
    torch.cuda.empty_cache()
    return out


def compressed_bytes(info):
    return info["file_bytes"] - 2 * (info["padded_words"] - info["total_words"])


def run_c4(args):
    import math

    import numpy as np
    import torch

    import paper_2601_22787_amd as eq
    import synth
    from synth.configs import config_matrices

    eq.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    specs = config_matrices(4)
    fmt = FORMATS[args.base_format]
    kernel_names = KERNEL if fmt == 1 else KERNEL_INT8
    layers = build_layers(eq, synth, specs, args.copies, dev, fmt, v2_copies=args.copies,
                          row_order=args.row_order, v2_rows=args.v2_tile_rows)
    ops = ["bf16", "gemv1", "gemv8"]
    copies = args.copies

    # device buffers shared by all steps
    wouts = [torch.empty(spec.params, dtype=torch.int16, device=dev) for spec in specs]
    codes_out = torch.empty(max(s.params for s in specs), dtype=torch.uint8, device=dev)
    bufs = []
    for item in layers:
        spec = item["spec"]
        d = {}
        for B in (1, 8):
            x = torch.from_numpy(synth.activations(spec, B).view(np.int16)).to(dev)
            y = torch.empty(B, spec.rows, dtype=torch.float32, device=dev)
            d[B] = (x, y, item["layers"][0].workspace(B), item["layers2"][0].workspace(B))
        bufs.append(d)
    infos = [blob_info(item["blob"]) for item in layers]
    infos2 = [blob_info(item["blob2"]) for item in layers]
    ALL = -1  # launch covering both matrices

    # One step: the layer's two matrices decoded to BF16 by one block-wise
    # launch (they are decompressed together, as a block's weights are),
    # then the fused GEMVs of each matrix at B = 1 and B = 8 (the two
    # matrices read different inputs, so they are separate launches).  Every
    # read of a matrix takes the next of its device copies (read k of step s:
    # copy (3 s + k) mod copies), so no launch finds its container in the
    # MALL from the launch before.
    reads = 3
    period = copies // math.gcd(reads, copies)

    def launches(s):
        def lay(item, k):
            return item["layers"][(reads * s + k) % copies]
        yield ALL, "bf16", lambda: eq.eq_decode_bf16_multi([lay(it, 0) for it in layers], wouts)
        for mi, item in enumerate(layers):
            for k, op in ((1, "gemv1"), (2, "gemv8")):
                B = 1 if op == "gemv1" else 8
                x, y, ws, _ = bufs[mi][B]
                L = lay(item, k)
                yield mi, op, (lambda L=L, x=x, B=B, y=y, ws=ws:
                               eq.eq_decode_gemv(L, x, B, None, y, ws))

    def one_step(s, timers=None):
        for mi, op, fn in launches(s):
            if timers is None:
                fn()
            else:
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
                fn()
                e1.record()
                timers.append((mi, op, e0, e1))

    # Reference: a plain elementwise copy of 256 MiB (uint8 to int8, so that
    # it runs as torch's copy kernel rather than a runtime blit shared with
    # the uploads), the known-size kernel against which HBM byte counters are
    # calibrated.
    ref_src = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
    ref_dst = torch.empty(256 << 20, dtype=torch.int8, device=dev)
    ref_dst.copy_(ref_src)
    c0 = torch.cuda.Event(enable_timing=True)
    c1 = torch.cuda.Event(enable_timing=True)
    c0.record()
    ref_dst.copy_(ref_src)
    c1.record()
    torch.cuda.synchronize()
    copy_gbs = 2 * ref_src.numel() / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del ref_src, ref_dst
    hbm_ref = hbm_reference(torch, dev)

    def check_status():
        for item in layers:
            for L in item["layers"] + item["layers2"]:
                rc = eq.eq_get_status(L)
                if rc != eq.EQ_OK:
                    raise RuntimeError(f"decode status {eq.eq_strerror(rc)}")

    for s in range(args.warmup):
        one_step(s)
    torch.cuda.synchronize()
    check_status()

    # The step as a serving loop would run it: one HIP graph per position in
    # the copy rotation (the library's calls only launch kernels, so they
    # capture), replayed in order.  Per-launch figures come from each op's
    # launches replayed as a graph of their own, and from an eager pass.
    graphs = []
    if not args.eager:
        for c in range(period):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                one_step(c)
            graphs.append(g)
        for c in range(period):
            graphs[c].replay()
    timers = []
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record()
    for s in range(args.steps):
        if graphs:
            graphs[(args.warmup + s) % period].replay()
        else:
            one_step(args.warmup + s, timers)
    t_end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = t_start.elapsed_time(t_end)
    ms_per_step = total_ms / args.steps
    if graphs:
        for s in range(args.steps):
            one_step(args.warmup + s, timers)
        torch.cuda.synchronize()
    check_status()

    per = {}
    for mi, op, e0, e1 in timers:
        per.setdefault((mi, op), []).append(e0.elapsed_time(e1))
    # GPU time per launch: each op's launches over the copy rotation,
    # captured back to back in a HIP graph (the eager figures above also
    # hold the host's launch and event gaps)
    per_graph = {}
    if not args.eager:
        fns = {}
        for c in range(period):
            for mi, op, fn in launches(c):
                fns.setdefault((mi, op), []).append(fn)
        for key, fl in fns.items():
            per_graph[key] = time_graph(lambda i, fl=fl: fl[i](), len(fl), 3)
    mats = list(range(len(specs)))
    kernels, fam = {}, {}
    for (mi, op), ts in per.items():
        covered = mats if mi == ALL else [mi]
        name = "layer" if mi == ALL else specs[mi].name
        B = 8 if op == "gemv8" else 1
        us_eager = 1000.0 * sum(ts) / len(ts)
        us = per_graph.get((mi, op), us_eager)
        q10, q50, q90 = (1000.0 * float(v) for v in np.percentile(ts, [10, 50, 90]))
        params = sum(specs[m].params for m in covered)
        nbytes = sum(algorithmic_bytes(infos[m], op, B) for m in covered)
        comp = sum(compressed_bytes(infos[m]) for m in covered)
        kernels[f"{name}.{op}"] = {
            "kernel": kernel_names[op], "us": round(us, 2), "us_eager": round(us_eager, 2),
            "us_eager_p10": round(q10, 2), "us_eager_p50": round(q50, 2),
            "us_eager_p90": round(q90, 2), "params": params,
            "gparams_per_s": round(params / us / 1e3, 1),
            "alg_bytes": nbytes, "gbs": round(nbytes / us / 1e3, 1),
            "hbm_frac": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4),
            "hbm_frac_compressed": round(comp / us / 1e3 / HBM_PEAK_GBS, 4)}
        f = fam.setdefault(op, {"us": 0.0, "launches": 0, "bytes": 0, "params": 0})
        f["us"] += us
        f["launches"] += 1
        f["bytes"] += nbytes
        f["params"] += params
    # dominant kernel: the op family with the largest share of the step;
    # figures per launch (mean over the family's launches)
    dom = max(fam, key=lambda k: fam[k]["us"])
    fd = fam[dom]
    dom_us = fd["us"] / fd["launches"]
    dom_bytes = fd["bytes"] / fd["launches"]
    achieved_gbs = fd["bytes"] / fd["us"] / 1e3

    # Container version 2 (tiles of 256 x 256, one phrase of 1-4 codes per
    # state update) of the same codes: every op timed launch by launch over
    # the rotated copies.
    v2 = {}
    for mi, item in enumerate(layers):
        spec, L2 = item["spec"], item["layers2"]
        out = wouts[mi]
        fns = {"gemv1": lambda i, mi=mi, L2=L2: eq.eq_decode_gemv(
                   L2[i % copies], bufs[mi][1][0], 1, None, bufs[mi][1][1], bufs[mi][1][3]),
               "gemv8": lambda i, mi=mi, L2=L2: eq.eq_decode_gemv(
                   L2[i % copies], bufs[mi][8][0], 8, None, bufs[mi][8][1], bufs[mi][8][3]),
               "bf16": lambda i, L2=L2, out=out: eq.eq_decode_bf16(L2[i % copies], out),
               "codes": lambda i, L2=L2, n=spec.params: eq.eq_decode_codes(
                   L2[i % copies], codes_out[:n])}
        for op, fn in fns.items():
            for i in range(args.warmup):
                fn(i)
            us_eager, p50, _ = time_eager(fn, copies, max(args.steps, 20))
            us = us_eager if args.eager else time_graph(fn, copies, 3)
            B = 8 if op == "gemv8" else 1
            nbytes = (algorithmic_bytes(infos2[mi], op, B) if op != "codes"
                      else compressed_bytes(infos2[mi]) + spec.params)
            v2[f"{spec.name}.{op}"] = {
                "kernel": V2_KERNEL[op], "us": round(us, 2), "us_eager": round(us_eager, 2),
                "us_eager_p50": round(p50, 2),
                "gparams_per_s": round(spec.params / us / 1e3, 1), "alg_bytes": nbytes,
                "hbm_frac": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4),
                "hbm_frac_compressed": round(compressed_bytes(infos2[mi]) / us / 1e3 /
                                             HBM_PEAK_GBS, 4)}
    check_status()

    # The target row: fused decode-GEMV at batch 1 on the 8192x28672 matrix,
    # compressed bytes over the launch time against the HBM peak.
    tr = {}
    for version, info, us in ((1, infos[0], kernels["down.gemv1"]["us"]),
                              (2, infos2[0], v2["down.gemv1"]["us"])):
        cb = compressed_bytes(info)
        tr[str(version)] = {"us": us, "compressed_bytes": cb,
                            "bits_per_param": round(8 * info["file_bytes"] / specs[0].params, 4),
                            "gbs": round(cb / us / 1e3, 1),
                            "frac": round(cb / us / 1e3 / HBM_PEAK_GBS, 4)}
    best = min(tr, key=lambda k: tr[k]["us"])
    target_row = {"shape": [specs[0].rows, specs[0].cols], "op": "fused decode-GEMV, batch 1",
                  "container": int(best), "kernel": (V2_KERNEL["gemv1"] if best == "2"
                                                     else kernel_names["gemv1"]),
                  "us": tr[best]["us"], "frac": tr[best]["frac"], "target_frac": TARGET_FRAC,
                  "entropy_bits": round(infos[0]["entropy"], 4), "by_container": tr}
    tc = kernel_counters(target_row["kernel"])
    target_row["traffic"] = tc.get("hbm_bytes") if tc else None
    if tc and "valu_insts" in tc:
        target_row["valu_lane_ops_per_param"] = round(64.0 * tc["valu_insts"] / specs[0].params,
                                                      2)

    params_per_step = sum(s.params for s in specs) * len(ops)
    value = params_per_step / (ms_per_step * 1e-3) / 1e9
    counters = kernel_counters(kernel_names[dom])
    result = {
        "metric": "decoded Gparams/s (decode->BF16 + fused decode-GEMV B=1,8 over the "
                  "8192x28672 and 28672x8192 layers); per-kernel us/layer and % HBM roofline",
        "value": round(value, 2), "unit": "Gparams/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u32", "data": "synthetic",
        "config": {"workload": f"Llama-70B MLP layers 8192x28672 + 28672x8192, "
                               f"{args.base_format.upper()} at ~2.0 "
                               "bits/param, 65536-symbol chunks, 256 rANS lanes/chunk "
                               "(container version 1); per step: both matrices decoded to BF16 "
                               "by one block-wise launch, then fused decode-GEMV B=1 and B=8 per "
                               "matrix",
                   "base_format": args.base_format,
                   "entropy_bits": [round(i["entropy"], 4) for i in infos],
                   "container_mb": [round(i["file_bytes"] / 1e6, 2) for i in infos],
                   "container_v2_mb": [round(i["file_bytes"] / 1e6, 2) for i in infos2],
                   "v2_tiles": [[i["lanes"], i["tile_cols"]] for i in infos2],
                   "v2_row_order": bool(args.row_order),
                   "copies_rotated": copies,
                   "launch": "eager" if args.eager else "HIP graphs of the step"},
        "roofline": {"bound": "hbm", "kernel": kernel_names[dom], "op": dom,
                     "achieved": round(achieved_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved_gbs / HBM_PEAK_GBS, 4),
                     "traffic": counters.get("hbm_bytes") if counters else None,
                     "alg_bytes": round(dom_bytes), "us_per_launch": round(dom_us, 2)},
        "target_row": target_row,
        "kernels": kernels,
        "container_v2": v2,
        "calibration_copy_gbs": round(copy_gbs, 1),
        "hbm_reference": hbm_ref,
        "wall_s_timed": round(wall, 3),
        "env": run_env(),
    }
    if counters and "valu_insts" in counters:
        # secondary: vector-ALU issue of the dominant kernel from its measured
        # SQ_INSTS_VALU (wave instructions, 64 lanes each) per launch
        lane_ops = 64.0 * counters["valu_insts"]
        result["roofline"]["alu"] = {
            "lane_ops_per_param": round(lane_ops / (fd["params"] / fd["launches"]), 2),
            "achieved_tops": round(lane_ops / dom_us / 1e6, 2), "peak_tops": round(ALU_PEAK_TOPS, 2),
            "frac": round(lane_ops / dom_us / 1e6 / ALU_PEAK_TOPS, 4)}
    if not args.no_cpu_baseline:
        threads = args.cpu_threads or min(16, os.cpu_count() or 1)
        result["cpu_baseline"] = cpu_baseline(layers, args.cpu_seconds, threads, fmt)
    print(json.dumps(result), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: runs on one GPU only; --gpus {args.gpus} is not supported (several "
              f"GPUs would each hold and decode their own output rows of every layer)",
              file=sys.stderr)
        sys.exit(2)
    if args.counters_from:
        summarise_counters(args.counters_from)
    elif args.workload == "c5":
        run_stack(args)
    elif args.workload == "prefill":
        run_prefill(args)
    elif args.workload == "c123":
        run_small(args)
    else:
        run_c4(args)


if __name__ == "__main__":
    main()
