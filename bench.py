#!/usr/bin/env python3
"""One-GPU benchmark of the AWSRC codec hot path on MI355X.

A step is one pass of the whole path over one synthetic module set already
resident in HBM: RTN-INT4 backbone, encoder seed search over all tiles and
seeds, gain ranking + serialization under the byte budget, and decode-add of
the resulting stream onto W0.  Prints one JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload down3b]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "encoded tile-seed candidates/sec + decode-add GB/s (fraction of roofline), 1 GPU"
PEAK_HBM_GBS = 8000.0            # MI355X HBM3E
PEAK_VALU_TOPS = 78.6            # fp32 vector lane-ops/s (157.3 TFLOP/s counting FMA as 2)
PEAK_MFMA_BF16_TFLOPS = 2500.0   # dense bf16 matrix-core flops/s


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# HBM bytes per launch measured with rocprofv3 --pmc FETCH_SIZE and WRITE_SIZE
# (one pass each; profiles/counters_*.md).  FETCH_SIZE is scaled by 2.0 and
# WRITE_SIZE by 1.0: the ratios of a 1 GiB device copy's bytes to what the
# same counters read for it.  An entry holds for the kernel sources it was
# measured on (SHA-256 over the listed files); after any change to them the
# figure is reported as null until the counters are taken again.
MEASURED_TRAFFIC = {
    ("encode", "down3b"): {
        "files": ["awsrc_internal.h", "basis.hip", "encode.hip", "encode_mfma.hip", "rescore64.h"],
        "sha256": "f62d25be5634403723df27196df17c023950b2ae27656e65a4a7f591ca919ee0",
        "bytes": 312266468},
    ("backbone", "down3b"): {
        "files": ["awsrc_internal.h", "backbone.hip"],
        "sha256": "45a13fcf353eda08999bbf4cb013c9277bb8ed2b76de5fa4ba077fa5d04cd960",
        "bytes": 147301701},
    ("decode_apply", "down3b"): {
        "files": ["awsrc_internal.h", "decode.hip"],
        "sha256": "057b327e7fba35e628bae904c069085ca5b059d365549ba26d800a9201b58c27",
        "bytes": 22875478},
    # the stack3b stream at 0.32 bpw of the at-scale measurement
    ("decode_apply", "stack3b@0.32"): {
        "files": ["awsrc_internal.h", "decode.hip"],
        "sha256": "057b327e7fba35e628bae904c069085ca5b059d365549ba26d800a9201b58c27",
        "bytes": 5037000000},
    # the whole reconstruction call: tile ordering (scans, copy) and the streaming pass
    ("reconstruct_bf16", "stack3b@0.32"): {
        "files": ["awsrc_internal.h", "decode.hip"],
        "sha256": "057b327e7fba35e628bae904c069085ca5b059d365549ba26d800a9201b58c27",
        "bytes": 9336000000},
}


def measured_traffic(kernel: str, workload: str):
    import hashlib

    e = MEASURED_TRAFFIC.get((kernel, workload))
    if e is None:
        return None
    h = hashlib.sha256()
    for f in e["files"]:
        with open(os.path.join(ROOT, "paper_2608_23144_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return e["bytes"] if h.hexdigest() == e["sha256"] else None


def ops_per_candidate(C: int, P: int, per_element: bool, gen_version: int = 1) -> float:
    """Algorithmic fp32 operations per (tile, seed): projection (cheapest of the
    direct P*C form and a length-C fast Walsh-Hadamard transform), solve with a
    precomputed factor, quantization and the coefficient-space score; per-element
    weights add the Gram gather and a P x P Cholesky factorization, and with the
    seeded coordinate permutation (generator version 2) also the transform of
    the permuted weights that the Gram gather then reads."""
    proj = min(P * C, C * int(math.log2(C)))
    ops = proj + 2 * P * P + 6 * P + 9
    if per_element:
        ops += P * (P + 1) / 2 + P ** 3 / 6 + P * P / 2 + P / 3
        if gen_version != 1:
            ops += C * int(math.log2(C))
    return float(ops)


def _oracle_chunk(job):
    """Worker of cpu_baseline: the oracle's encoder on one chunk of tiles, one
    thread; returns the compute time."""
    R, D, op = job
    from threadpoolctl import threadpool_limits

    from oracle import awsrc_oracle as O

    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
        O.encode_tiles(R, D, op)
        return time.perf_counter() - t0


def _oracle_warm(job):
    """Pool initializer: imports and one small call, so that every worker is
    warm before the timed map."""
    _oracle_chunk(job)


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, inputs, seconds: float):
    """The oracle as it stands, on a bounded sample of the same workload's
    tiles, over worker processes (one thread each) that take contiguous
    chunks of tiles: a pilot sizes the sample at about 2 x `seconds` of CPU
    work in all, and the rate is the sample's candidates over the timed
    map's wall time (the workers are started and warmed first)."""
    import multiprocessing as mp

    from oracle import awsrc_oracle as O

    m = wl.modules[0]
    W32 = inputs[0]["W32"].cpu().numpy()
    d = inputs[0]["d"].cpu().numpy()
    op = O.Params(C=wl.C, P=wl.P, b=wl.b, S=wl.S, basis_key=wl.basis_key, ridge_lambda=wl.ridge_lambda,
                  idx_bits=wl.idx_bits)
    _, _, _, W0o = O.rtn_backbone(W32)
    R = O.tiles(O.residual(W32, W0o), wl.C)
    D = O.tile_weights(d, m.rows, m.cols, wl.C)
    # the host's CPU share for one GPU is 16 cores, whatever the affinity mask shows
    nproc = max(1, min(16, len(os.sched_getaffinity(0))))
    # pilot in this process: per-tile time (the oracle also pays a fixed cost per call)
    _oracle_chunk((R[:64], D[:64], op))
    t1 = _oracle_chunk((R[:64], D[:64], op))
    t2 = _oracle_chunk((R[:256], D[:256], op))
    per_tile = max((t2 - t1) / 192, 1e-6)
    per = int(max(256, 2.0 * seconds / nproc / per_tile))
    n2 = int(min(R.shape[0], per * nproc))
    per = -(-n2 // nproc)
    jobs = [(R[i:i + per], D[i:i + per], op) for i in range(0, n2, per)]
    ctx = mp.get_context("spawn")  # fresh interpreters: nothing of this process's GPU state
    with ctx.Pool(nproc, initializer=_oracle_warm, initargs=((R[:16], D[:16], op),)) as pool:
        pool.map(_oracle_chunk, [(R[:16], D[:16], op)] * nproc, chunksize=1)  # all started
        t0 = time.perf_counter()
        pool.map(_oracle_chunk, jobs, chunksize=1)
        dt = time.perf_counter() - t0
    return {"value": n2 * wl.S / dt, "unit": "candidates/s", "cores": nproc, "kind": "oracle",
            "cpu": _cpu_model(),
            "sample": f"first {n2} of {R.shape[0]} tiles of {m.name} ({m.rows}x{m.cols}), all {wl.S} seeds, "
                      f"fp64 numpy, {len(jobs)} chunks over {nproc} worker processes of 1 thread, "
                      f"{dt:.1f} s wall"}


def decode_at_scale(awsrc, torch, name: str, bpw: float, reps: int):
    """Decode-add of a large stream: records drawn at random for every tile of
    the named workload (all gains positive), ranked globally at `bpw`, then
    applied `reps` times onto fp32 W0 buffers of the workload's shapes (an
    add onto the same tiles each time).  Timed with HIP events on the
    library's stream around the apply launches only."""
    from synth import gen_records, workload

    wl = workload(name)
    dev = torch.device("cuda:0")
    shapes = [(m.rows, m.cols) for m in wl.modules]
    p = awsrc.make_params(wl.C, wl.P, wl.b, wl.S, basis_key=wl.basis_key, ridge_lambda=wl.ridge_lambda,
                          idx_bits=wl.idx_bits)
    rec = gen_records(wl.n_tiles, wl.P, wl.b, wl.S, seed=4242, device=dev, frac_nonpositive=0.0, frac_ties=0.0)
    s, K, _ = awsrc.awsrc_rank_prefix(p, shapes, awsrc.AWSRC_MODE_GLOBAL, bpw, rec["seed"], rec["codes"],
                                      rec["scale"], rec["gain"])
    del rec
    W0 = [torch.zeros(r, c, dtype=torch.float32, device=dev) for r, c in shapes]
    plan, dws = awsrc.awsrc_decode_prepare(s, W0)
    stream = torch.cuda.current_stream()
    awsrc.awsrc_decode_apply(plan)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        awsrc.awsrc_decode_apply(plan)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    nbytes = K * (plan.L_rec + 2 * wl.C * 4)
    gbs = nbytes / (ms / 1e3) / 1e9
    del W0, plan, dws
    rec_stats = reconstruct_at_scale(awsrc, torch, wl, shapes, s, K, reps, bpw)
    del s
    # device-copy ceiling: one large copy, read + write bytes
    n = 1 << 30
    x = torch.empty(n, dtype=torch.float32, device=dev)
    y = torch.empty_like(x)
    y.copy_(x)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(3):
        y.copy_(x)
    e1.record(stream)
    torch.cuda.synchronize()
    copy_gbs = 3 * 2 * 4 * n / (e0.elapsed_time(e1) / 1e3) / 1e9
    del x, y
    torch.cuda.empty_cache()
    rec_stats["frac_copy"] = rec_stats["GB/s"] / copy_gbs
    return {"workload": f"{name} stream at {bpw} bpw, fp32 W0", "modules": len(shapes), "records": K,
            "bytes": nbytes, "ms": ms, "GB/s": gbs, "frac_hbm": gbs / PEAK_HBM_GBS,
            "copy_GB/s": copy_gbs, "frac_copy": gbs / copy_gbs,
            "traffic": measured_traffic("decode_apply", f"{name}@{bpw}"), "reconstruct_bf16": rec_stats}


def reconstruct_at_scale(awsrc, torch, wl, shapes, s, K, reps, bpw):
    """Dense bf16 reconstruction of every module from a random RTN backbone
    (codes, fp16 scales in [1e-3, 2e-3), zero points) plus the stream `s`.
    Algorithmic bytes: codes (1/2 B per weight), scale and zero (3 B per
    group of 128), the records, and the bf16 output (2 B per weight).  Each
    call synchronizes once before its two launches, and the timed region
    (HIP events on the library's stream) includes that host round trip."""
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(77)
    bbs = []
    for r, c in shapes:
        codes = torch.randint(0, 256, (r, c // 2), dtype=torch.uint8, device=dev, generator=g)
        sc = (torch.rand(r, c // 128, device=dev, generator=g) * 1e-3 + 1e-3).to(torch.float16).view(torch.int16)
        z = torch.randint(0, 16, (r, c // 128), dtype=torch.uint8, device=dev, generator=g)
        bbs.append((codes, sc, z))
    outs = [torch.empty(r, c, dtype=torch.bfloat16, device=dev) for r, c in shapes]
    plan, ws = awsrc.awsrc_decode_prepare(s, outs)
    stream = torch.cuda.current_stream()
    awsrc.awsrc_reconstruct_bf16(plan, bbs, 128)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        awsrc.awsrc_reconstruct_bf16(plan, bbs, 128)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    n_w = sum(r * c for r, c in shapes)
    nbytes = n_w // 2 + 3 * (n_w // 128) + K * plan.L_rec + 2 * n_w
    del outs, bbs, plan, ws
    torch.cuda.empty_cache()
    gbs = nbytes / (ms / 1e3) / 1e9
    return {"weights": n_w, "bytes": nbytes, "ms": ms, "GB/s": gbs, "frac_hbm": gbs / PEAK_HBM_GBS,
            "traffic": measured_traffic("reconstruct_bf16", f"{wl.name}@{bpw}")}


def mfma_screen(C: int, P: int, per_element: bool, gen_version: int) -> bool:
    """The encoder's matrix-core screen runs (projection as exact bf16 x 3 products)."""
    if P > 8 or (per_element and gen_version != 1):
        return False
    return C == 64 or (C == 128 and not per_element)


def bound_ops_per_candidate(P: int) -> float:
    """Vector work of the pruning bound per candidate: the forward solve with the
    unit lower factor (P(P-1)/2), sum of w_p^2 / e_p (2P) and the comparison."""
    return P * (P - 1) / 2 + 2 * P + 1


def encode_split_bound(C: int, P: int, per_element: bool, gen_version: int, scored_frac: float) -> dict:
    """Split roofline of the encoder with the projection on the matrix cores:
    6 P C bf16 flops per candidate there (three exact bf16 parts of fp32 u),
    and on the vector ALUs the post-projection work: every candidate's bound
    plus, for the fraction scored in full, the rest of the unpruned count
    (ops_per_candidate less the projection).  Without pruning the fraction is 1."""
    proj = min(P * C, C * int(math.log2(C)))
    full = ops_per_candidate(C, P, per_element, gen_version) - proj
    bnd = bound_ops_per_candidate(P)
    valu = bnd + scored_frac * (full - bnd) if scored_frac < 1.0 else full
    return {"mfma_flops_per_candidate": 6.0 * P * C, "valu_ops_per_candidate": valu}


def sdq_timing(awsrc, torch, wl, bb, stream, reps: int = 20) -> dict:
    """RTN-INT4-SDQ backbone (Sec. 3.3, Sec. 4): SDQ of the step's group scales
    and W0 with the dequantized scales, timed with HIP events (outside the
    step; the step's encoder repairs the RTN-v1 backbone).  Algorithmic bytes:
    encode 2 B read + 1 B written per group and 8 B per block of 256; W0 0.5 B
    of codes read and 4 B written per weight, 2 B (zero point, code) per group
    and 8 B per block."""
    n_w = sum(b[0].numel() * 2 for b in bb)
    n_g = sum(b[1].numel() for b in bb)
    n_blk = sum((b[1].numel() + 255) // 256 for b in bb)
    sdqs = [awsrc.awsrc_sdq_encode(b[1]) for b in bb]
    outs = [awsrc.awsrc_backbone_sdq_dequant(b[0], b[2], q) for b, q in zip(bb, sdqs)]
    e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    torch.cuda.synchronize()
    e[0].record(stream)
    for _ in range(reps):
        for b in bb:
            awsrc.awsrc_sdq_encode(b[1])
    e[1].record(stream)
    for _ in range(reps):
        for b, q, o in zip(bb, sdqs, outs):
            awsrc.awsrc_backbone_sdq_dequant(b[0], b[2], q, out=o)
    e[2].record(stream)
    torch.cuda.synchronize()
    enc_ms = e[0].elapsed_time(e[1]) / reps
    deq_ms = e[1].elapsed_time(e[2]) / reps
    enc_bytes = 3 * n_g + 8 * n_blk
    deq_bytes = n_w // 2 + 4 * n_w + 2 * n_g + 8 * n_blk
    return {"groups": n_g, "scale_bits_per_weight": (8 * n_g + 64 * n_blk) / n_w,
            "fp16_scale_bits_per_weight": 16 * n_g / n_w,
            "encode_ms": enc_ms, "dequant_ms": deq_ms, "dequant_bytes": deq_bytes,
            "dequant_GB/s": deq_bytes / (deq_ms / 1e3) / 1e9,
            "dequant_frac_hbm": deq_bytes / (deq_ms / 1e3) / 1e9 / PEAK_HBM_GBS,
            "encode_bytes": enc_bytes}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="down3b")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--decode-workload", default="stack3b",
                    help="workload whose shapes size the at-scale decode-add measurement ('' to skip)")
    ap.add_argument("--decode-bpw", type=float, default=0.32)
    ap.add_argument("--gen-version", type=int, default=1, choices=(1, 2),
                    help="basis generator version (2 adds the seeded coordinate permutation)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run three plain 1 GiB device copies (the known-size kernel that "
                         "scales the HBM byte counters) and exit")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        log("bench.py measures a single GPU: the codec has no cross-GPU step "
            "(run with --gpus 1)")
        return 2

    import torch

    if args.copy_calibration:
        n = 1 << 28  # 2^28 floats = 1 GiB per buffer
        x = torch.ones(n, dtype=torch.float32, device="cuda")
        y = torch.empty_like(x)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        log(f"[bench] copied 3 x {4 * n} bytes")
        return 0

    import paper_2608_23144_amd as awsrc
    from synth import gen_module_inputs, workload

    wl = workload(args.workload)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    p = awsrc.make_params(wl.C, wl.P, wl.b, wl.S, basis_key=wl.basis_key, ridge_lambda=wl.ridge_lambda,
                          idx_bits=wl.idx_bits, gen_version=args.gen_version)
    mods = wl.modules
    log(f"[bench] workload {wl.name}: {len(mods)} module(s), {wl.n_weights} weights, T={wl.n_tiles}, S={wl.S}")
    inputs = [gen_module_inputs(wl, m, dev) for m in mods]
    T = wl.n_tiles
    seed = torch.empty(T, dtype=torch.int16, device=dev)
    codes = torch.empty(T, wl.P, dtype=torch.int8, device=dev)
    scale = torch.empty(T, dtype=torch.int16, device=dev)
    gain = torch.empty(T, dtype=torch.float64, device=dev)
    bb, enc_out, ws = [], [], []
    off = 0
    for m, inp in zip(mods, inputs):
        t_m = m.rows * m.cols // wl.C
        bb.append((torch.empty(m.rows, m.cols // 2, dtype=torch.uint8, device=dev),
                   torch.empty(m.rows, m.cols // 128, dtype=torch.int16, device=dev),
                   torch.empty(m.rows, m.cols // 128, dtype=torch.uint8, device=dev),
                   torch.empty(m.rows, m.cols, dtype=torch.float32, device=dev)))
        enc_out.append({"seed": seed[off:off + t_m], "codes": codes[off:off + t_m], "scale": scale[off:off + t_m],
                        "gain": gain[off:off + t_m], "alpha": None})
        d_mode = awsrc.AWSRC_D_PER_COL if inp["d"].dim() == 1 else awsrc.AWSRC_D_PER_ELEM
        ws.append(torch.empty(awsrc.encode_workspace_bytes(p, inp["W"], d_mode), dtype=torch.uint8, device=dev))
        off += t_m
    shapes = [(m.rows, m.cols) for m in mods]
    mode = awsrc.AWSRC_MODE_GLOBAL if wl.mode == "global" else awsrc.AWSRC_MODE_PER_MODULE
    bpw = max(wl.budgets)
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
    acc = {"backbone": 0.0, "encode": 0.0, "rank": 0.0, "decode_prepare": 0.0, "decode_apply": 0.0}
    last = {}

    def step(record: bool):
        ev[0].record(stream)
        for inp, b in zip(inputs, bb):
            awsrc.awsrc_backbone_rtn(inp["W"], out=b)
        ev[1].record(stream)
        for inp, b, e, w in zip(inputs, bb, enc_out, ws):
            awsrc.awsrc_encode_tiles(p, inp["W"], b[3], inp["d"], out=e, workspace=w)
        ev[2].record(stream)
        s, K, ne = awsrc.awsrc_rank_prefix(p, shapes, mode, bpw, seed, codes, scale, gain)
        ev[3].record(stream)
        plan, dws = awsrc.awsrc_decode_prepare(s, [b[3] for b in bb], workspace=last.get("dws"))
        ev[4].record(stream)
        awsrc.awsrc_decode_apply(plan)
        ev[5].record(stream)
        last.update(K=K, n_eligible=ne, stream_len=int(s.numel()), L=plan.L_rec, dws=dws)
        if record:
            torch.cuda.synchronize()
            for k, (a, b) in zip(acc, zip(ev[:-1], ev[1:])):
                acc[k] += a.elapsed_time(b)

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    log(f"[bench] warmup done ({args.warmup} steps); timing {args.steps} steps")
    # wall clock over exactly K steps; stage events are read after each step
    t_wall = 0.0
    for _ in range(args.steps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        step(True)
        t_wall += time.perf_counter() - t0
    ms_step = 1e3 * t_wall / args.steps
    stage_ms = {k: v / args.steps for k, v in acc.items()}
    cand = wl.candidates
    value = cand / (ms_step / 1e3)

    per_elem = wl.d_mode == "elem"
    opc = ops_per_candidate(wl.C, wl.P, per_elem, args.gen_version)
    enc_s = stage_ms["encode"] / 1e3
    # candidates scored in full by the last step's screens (the pruned screen
    # scores a data-dependent part; every other screen scores all)
    scored = sum(awsrc.awsrc_encode_scored(e) for e in enc_out)
    f_scored = scored / cand
    if mfma_screen(wl.C, wl.P, per_elem, args.gen_version):
        sb = encode_split_bound(wl.C, wl.P, per_elem, args.gen_version, f_scored)
        t_mfma = cand * sb["mfma_flops_per_candidate"] / (PEAK_MFMA_BF16_TFLOPS * 1e12)
        t_valu = cand * sb["valu_ops_per_candidate"] / (PEAK_VALU_TOPS * 1e12)
        if t_mfma >= t_valu:
            bound, unit, peak = "mfma", "TFLOP/s", PEAK_MFMA_BF16_TFLOPS
            achieved = cand * sb["mfma_flops_per_candidate"] / enc_s / 1e12
        else:
            bound, unit, peak = "alu", "Tops/s", PEAK_VALU_TOPS
            achieved = cand * sb["valu_ops_per_candidate"] / enc_s / 1e12
        split = dict(sb, scored_fraction=f_scored, t_mfma_ms=1e3 * t_mfma, t_valu_ms=1e3 * t_valu)
    else:
        bound, unit, peak = "alu", "Tops/s", PEAK_VALU_TOPS
        achieved = cand * opc / enc_s / 1e12
        split = {"scored_fraction": f_scored}
    K, L = last["K"], last["L"]
    dec_bytes = K * (L + 2 * wl.C * 4)
    dec_gbs = dec_bytes / (stage_ms["decode_apply"] / 1e3) / 1e9 if stage_ms["decode_apply"] > 0 else None
    n_groups = wl.n_weights // 128
    bb_bytes = wl.n_weights * (2 if wl.w_dtype == "bf16" else 4) + wl.n_weights // 2 + 3 * n_groups + 4 * wl.n_weights
    bb_gbs = bb_bytes / (stage_ms["backbone"] / 1e3) / 1e9

    out = {
        "metric": METRIC, "value": value, "unit": "candidates/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": wl.name, "modules": [f"{r}x{c}" for r, c in shapes], "C": wl.C, "P": wl.P,
                   "b": wl.b, "S": wl.S, "weights": wl.d_mode, "mode": wl.mode, "bpw": bpw, "tiles": T,
                   "candidates": cand, "generator": args.gen_version},
        "roofline": {"bound": bound, "kernel": "awsrc_encode_tiles (basis, factors, screen, fp64 re-score)",
                     "achieved": achieved, "peak": peak, "unit": unit, "frac": achieved / peak,
                     "traffic": measured_traffic("encode", wl.name) if args.gen_version == 1 else None,
                     "traffic_unit": "bytes per launch", "split": split,
                     "ops_per_candidate_unpruned": opc},
        "encode_candidates_per_s": cand / enc_s,
        "decode_add": {"records": K, "bytes": dec_bytes, "ms": stage_ms["decode_apply"], "GB/s": dec_gbs,
                       "frac_hbm": (dec_gbs / PEAK_HBM_GBS) if dec_gbs else None,
                       "traffic": measured_traffic("decode_apply", wl.name)},
        "backbone": {"bytes": bb_bytes, "ms": stage_ms["backbone"], "GB/s": bb_gbs, "frac_hbm": bb_gbs / PEAK_HBM_GBS,
                     "traffic": measured_traffic("backbone", wl.name)},
        "stage_ms": stage_ms,
        "stream": {"K": K, "n_eligible": last["n_eligible"], "bytes": last["stream_len"], "L_rec": L},
        "device": torch.cuda.get_device_name(0),
    }
    out["backbone_sdq"] = sdq_timing(awsrc, torch, wl, bb, stream)
    del inputs, bb, enc_out, ws
    torch.cuda.empty_cache()
    if args.decode_workload:
        log(f"[bench] decode-add at scale: {args.decode_workload} at {args.decode_bpw} bpw")
        out["decode_add_at_scale"] = decode_at_scale(awsrc, torch, args.decode_workload, args.decode_bpw, 5)
    if not args.no_cpu_baseline:
        wl_inputs = [gen_module_inputs(wl, m, dev) for m in mods[:1]]
        log("[bench] timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(wl, wl_inputs, args.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
