#!/usr/bin/env python3
"""One-GPU benchmark of the AWSRC codec hot path on MI355X.

A step is one pass of the whole path over one synthetic workload already
resident in HBM (by default the 36-layer 3B stack: 252 modules, 2.77G
weights, 43.35M tiles, S = 512 seeds): RTN-INT4 backbone of every module,
the encoder's seed search over every tile and seed, one global gain ranking
with serialization at the largest byte budget, decode-add of that stream onto
W0, and every smaller budget's prefix of the same stream decoded (dense bf16)
without re-encoding.  Smaller workloads are timed after it and reported under
"extra"; the oracle's rate on a bounded row sample is "cpu_baseline".  Prints
one JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload stack3b]
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
UNPACKED_VALU_TOPS = 39.3        # the same without packed fp32 (one op per lane per cycle), which the build disables
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
    # one step of the 36-layer 3B stack (profiles/counters_stack3b.md): the
    # encode call over all 252 modules (screen 29.74 GB, fp64 re-score
    # 29.31 GB, tables), the 252 backbone launches, the decode-add of the
    # 0.32 bpw stream, the reconstruction of its four nested prefixes (tile
    # ordering and the streaming pass), and the same on the SDQ backbone
    ("encode", "stack3b"): {
        "files": ["awsrc_internal.h", "basis.hip", "encode.hip", "encode_mfma.hip", "encode_pe.hip",
                  "rescore_pe.hip", "rescore64.h"],
        "sha256": "f5cd199c3a5245c6611d36b08ee9fe96bce500bab8f26b718433d744bcd47246",
        "bytes": 59053364832},
    ("backbone", "stack3b"): {
        "files": ["awsrc_internal.h", "backbone.hip"],
        "sha256": "dd09c1f2caf969e853367c60ca0066165bb345dae7435d5e68306dc76e166f06",
        "bytes": 18135252320},
    ("decode_apply", "stack3b"): {
        "files": ["awsrc_internal.h", "decode.hip"],
        "sha256": "714d9fc777f576f347fc8ca0e18b6a2edc15cf7e84d2c2ff7b727c84c5f3c69c",
        "bytes": 5032715136},
    ("reconstruct_bf16", "stack3b"): {
        "files": ["awsrc_internal.h", "decode.hip"],
        "sha256": "714d9fc777f576f347fc8ca0e18b6a2edc15cf7e84d2c2ff7b727c84c5f3c69c",
        "bytes": 26212606368},
    ("reconstruct_bf16_sdq", "stack3b"): {
        "files": ["awsrc_internal.h", "decode.hip"],
        "sha256": "714d9fc777f576f347fc8ca0e18b6a2edc15cf7e84d2c2ff7b727c84c5f3c69c",
        "bytes": 26142208960},
    # one step of the 32B layer (profiles/counters_layer32b.md)
    ("encode", "layer32b"): {
        "files": ["awsrc_internal.h", "basis.hip", "encode.hip", "encode_mfma.hip", "encode_pe.hip",
                  "rescore_pe.hip", "rescore64.h"],
        "sha256": "f5cd199c3a5245c6611d36b08ee9fe96bce500bab8f26b718433d744bcd47246",
        "bytes": 8115737536},
    ("backbone", "layer32b"): {
        "files": ["awsrc_internal.h", "backbone.hip"],
        "sha256": "dd09c1f2caf969e853367c60ca0066165bb345dae7435d5e68306dc76e166f06",
        "bytes": 3185498720},
    ("decode_apply", "layer32b"): {
        "files": ["awsrc_internal.h", "decode.hip"],
        "sha256": "714d9fc777f576f347fc8ca0e18b6a2edc15cf7e84d2c2ff7b727c84c5f3c69c",
        "bytes": 951661440},
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


def cpu_baseline(wl, sample, seconds: float):
    """The oracle as it stands, on a bounded, deterministic sample of the same
    workload: every n-th row of every module (all of that row's tiles), with n
    the smallest power-of-two multiple of the collected row step whose tiles a
    pilot estimates at no more than about 2 x `seconds` of CPU work in all.
    Worker processes (one thread each) take contiguous chunks of tiles; the
    rate is the sample's candidates over the timed map's wall time (workers
    started and warmed first).  `sample` holds, per module, the fp32 weights
    and weights d of the collected rows (every `step`-th row)."""
    import multiprocessing as mp

    import numpy as np

    from oracle import awsrc_oracle as O

    op = O.Params(C=wl.C, P=wl.P, b=wl.b, S=wl.S, basis_key=wl.basis_key, ridge_lambda=wl.ridge_lambda,
                  idx_bits=wl.idx_bits)
    step0 = sample["step"]

    def tiles_at(k):
        Rs, Ds = [], []
        for m, (W32, d) in zip(wl.modules, sample["rows"]):
            W32 = W32[::k]
            dd = d if d.ndim == 1 else d[::k]
            _, _, _, W0o = O.rtn_backbone(W32)
            Rs.append(O.tiles(O.residual(W32, W0o), wl.C))
            Ds.append(O.tile_weights(dd, W32.shape[0], m.cols, wl.C))
        return np.concatenate(Rs), np.concatenate(Ds)

    # the host's CPU share for one GPU is 16 cores, whatever the affinity mask shows
    nproc = max(1, min(16, len(os.sched_getaffinity(0))))
    R1, D1 = tiles_at(1)
    # pilot in this process: per-tile time (the oracle also pays a fixed cost per call)
    _oracle_chunk((R1[:64], D1[:64], op))
    t1 = _oracle_chunk((R1[:64], D1[:64], op))
    t2 = _oracle_chunk((R1[:256], D1[:256], op))
    per_tile = max((t2 - t1) / 192, 1e-6)
    k = 1
    while R1.shape[0] / k * per_tile > 2.0 * seconds * nproc and k < 1 << 20:
        k *= 2
    R, D = (R1, D1) if k == 1 else tiles_at(k)
    n2 = R.shape[0]
    per = -(-n2 // (4 * nproc))
    jobs = [(R[i:i + per], D[i:i + per], op) for i in range(0, n2, per)]
    ctx = mp.get_context("spawn")  # fresh interpreters: nothing of this process's GPU state
    with ctx.Pool(nproc, initializer=_oracle_warm, initargs=((R[:16], D[:16], op),)) as pool:
        pool.map(_oracle_chunk, [(R[:16], D[:16], op)] * nproc, chunksize=1)  # all started
        t0 = time.perf_counter()
        pool.map(_oracle_chunk, jobs, chunksize=1)
        dt = time.perf_counter() - t0
    rate = n2 * wl.S / dt
    return {"value": rate, "unit": "candidates/s", "cores": nproc, "kind": "oracle", "cpu": _cpu_model(),
            "sample": f"every {step0 * k}th row of each of the {len(wl.modules)} modules of {wl.name} (all tiles "
                      f"of those rows): {n2} of {wl.n_tiles} tiles, all {wl.S} seeds, fp64 numpy, {len(jobs)} "
                      f"chunks over {nproc} worker processes of 1 thread, {dt:.1f} s wall",
            "extrapolated_full_encode_s": wl.candidates / rate}


def mfma_screen(C: int, P: int, per_element: bool, gen_version: int) -> bool:
    """The encoder's matrix-core screen runs (projection as exact bf16 x 3 products)."""
    if P > 8 or (per_element and gen_version != 1):
        return False
    return C == 64 or (C == 128 and not per_element)


def bound_ops_per_candidate(P: int, per_element: bool = False) -> float:
    """Vector work of the pruning bound per candidate: the forward solve with the
    unit lower factor (P(P-1)/2), sum of w_p^2 / e_p (2P) and the comparison;
    with per-element weights every candidate's factor comes first (the Gram
    gather and the P x P factorization)."""
    ops = P * (P - 1) / 2 + 2 * P + 1
    if per_element:
        ops += P * (P + 1) / 2 + P ** 3 / 6 + P * P / 2 + P / 3
    return ops


def encode_split_bound(C: int, P: int, per_element: bool, gen_version: int, scored_frac: float) -> dict:
    """Split roofline of the encoder with the projection on the matrix cores:
    6 P C bf16 flops per candidate there (three exact bf16 parts of fp32 u),
    and on the vector ALUs the post-projection work: every candidate's bound
    plus, for the fraction scored in full, the rest of the unpruned count
    (ops_per_candidate less the projection).  Without pruning the fraction is 1."""
    proj = min(P * C, C * int(math.log2(C)))
    full = ops_per_candidate(C, P, per_element, gen_version) - proj
    bnd = bound_ops_per_candidate(P, per_element)
    valu = bnd + scored_frac * (full - bnd) if scored_frac < 1.0 else full
    return {"mfma_flops_per_candidate": 6.0 * P * C, "valu_ops_per_candidate": valu}


def sdq_timing(awsrc, torch, wl, run, stream, reps: int = 20) -> dict:
    """RTN-INT4-SDQ backbone (Sec. 3.3, Sec. 4): SDQ of the step's group scales
    and W0 with the dequantized scales, and the dense bf16 reconstruction of
    the step's four prefixes on that backbone (the evaluation form Sec. 4
    uses), timed with HIP events (outside the step; the step's encoder
    repairs the RTN-v1 backbone).  Algorithmic bytes: encode 2 B read + 1 B
    written per group and 8 B per block of 256; W0 0.5 B of codes read and
    4 B written per weight, 2 B (zero point, code) per group and 8 B per
    block; reconstruction as the step's, with 2 B per group for the zero
    point and scale code and 8 B per block."""
    bb = run.bb
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
    rc = {}
    last = run.last
    if "plan" in last:
        sbb = [(b[0], b[2], q[0], q[1], q[2]) for b, q in zip(bb, sdqs)]
        ks = [kb for _, kb in last["prefixes"]]
        r_reps = 5
        awsrc.awsrc_reconstruct_bf16_sdq(last["plan"], sbb, K_out=ks, outs=run.outs)
        torch.cuda.synchronize()
        e[0].record(stream)
        for _ in range(r_reps):
            awsrc.awsrc_reconstruct_bf16_sdq(last["plan"], sbb, K_out=ks, outs=run.outs)
        e[1].record(stream)
        torch.cuda.synchronize()
        rc_ms = e[0].elapsed_time(e[1]) / r_reps
        rc_bytes = n_w // 2 + 2 * n_g + 8 * n_blk + len(ks) * 2 * n_w + max(ks) * run.L
        rc = {"reconstruct_prefixes": len(ks), "reconstruct_ms": rc_ms, "reconstruct_bytes": rc_bytes,
              "reconstruct_GB/s": rc_bytes / (rc_ms / 1e3) / 1e9,
              "reconstruct_frac_hbm": rc_bytes / (rc_ms / 1e3) / 1e9 / PEAK_HBM_GBS,
              "reconstruct_traffic": measured_traffic("reconstruct_bf16_sdq", wl.name)}
    return {**rc, "groups": n_g, "scale_bits_per_weight": (8 * n_g + 64 * n_blk) / n_w,
            "fp16_scale_bits_per_weight": 16 * n_g / n_w,
            "encode_ms": enc_ms, "dequant_ms": deq_ms, "dequant_bytes": deq_bytes,
            "dequant_GB/s": deq_bytes / (deq_ms / 1e3) / 1e9,
            "dequant_frac_hbm": deq_bytes / (deq_ms / 1e3) / 1e9 / PEAK_HBM_GBS,
            "encode_bytes": enc_bytes}


class Run:
    """One workload resident in HBM and the buffers of its step: inputs W
    (storage dtype) and d, the backbone (codes, scales, zero points, fp32 W0),
    the encoder's outputs concatenated in module order with its workspace (one
    awsrc_encode_modules call encodes every module), and bf16 buffers for the
    dense reconstructions (one set per budget)."""

    def __init__(self, awsrc, torch, wl, gen_version: int, dev, sample_step: int = 0):
        from synth import gen_module_inputs

        self.wl = wl
        self.p = awsrc.make_params(wl.C, wl.P, wl.b, wl.S, basis_key=wl.basis_key, ridge_lambda=wl.ridge_lambda,
                                   idx_bits=wl.idx_bits, gen_version=gen_version)
        self.shapes = [(m.rows, m.cols) for m in wl.modules]
        T = wl.n_tiles
        self.seed = torch.empty(T, dtype=torch.int16, device=dev)
        self.codes = torch.empty(T, wl.P, dtype=torch.int8, device=dev)
        self.scale = torch.empty(T, dtype=torch.int16, device=dev)
        self.gain = torch.empty(T, dtype=torch.float64, device=dev)
        self.inputs, self.bb = [], []
        self.sample = {"step": sample_step, "rows": []}
        off = 0
        for m in wl.modules:
            inp = gen_module_inputs(wl, m, dev)
            if sample_step:
                d = inp["d"] if inp["d"].dim() == 1 else inp["d"][::sample_step]
                self.sample["rows"].append((inp["W32"][::sample_step].cpu().numpy(), d.cpu().numpy()))
            del inp["W32"]
            self.inputs.append(inp)
            t_m = m.rows * m.cols // wl.C
            self.bb.append((torch.empty(m.rows, m.cols // 2, dtype=torch.uint8, device=dev),
                            torch.empty(m.rows, m.cols // 128, dtype=torch.int16, device=dev),
                            torch.empty(m.rows, m.cols // 128, dtype=torch.uint8, device=dev),
                            torch.empty(m.rows, m.cols, dtype=torch.float32, device=dev)))
            off += t_m
        self.enc_out = {"seed": self.seed, "codes": self.codes, "scale": self.scale, "gain": self.gain,
                        "alpha": None}
        d_mode = awsrc.AWSRC_D_PER_COL if wl.d_mode == "col" else awsrc.AWSRC_D_PER_ELEM
        w_dtype = awsrc.AWSRC_DTYPE_BF16 if wl.w_dtype == "bf16" else awsrc.AWSRC_DTYPE_F32
        self.ws = torch.empty(max(1, awsrc.encode_modules_workspace_bytes(self.p, self.shapes, w_dtype, d_mode)),
                              dtype=torch.uint8, device=dev)
        self.W_list = [inp["W"] for inp in self.inputs]
        self.d_list = [inp["d"] for inp in self.inputs]
        self.W0_list = [b[3] for b in self.bb]
        # one set of dense bf16 targets per budget (the nested prefixes are
        # reconstructed in one pass)
        self.outs = [[torch.empty(r, c, dtype=torch.bfloat16, device=dev) for r, c in self.shapes]
                     for _ in wl.budgets]
        self.mode = awsrc.AWSRC_MODE_GLOBAL if wl.mode == "global" else awsrc.AWSRC_MODE_PER_MODULE
        self.L = awsrc.awsrc_record_bytes(self.p, T)
        self.h = awsrc.awsrc_header_bytes(len(self.shapes))
        self.last = {}


STAGES = ("backbone", "encode", "rank", "decode_prepare", "decode_apply", "reconstruct")


def run_steps(awsrc, torch, run: Run, steps: int, warmup: int):
    """Time `steps` steps after `warmup` untimed ones.  A step: backbone of
    every module; encoder seed search of every module; one ranking at the
    largest budget; decode-add of that stream in place onto the fp32 W0
    (prepare = validation and tables, apply = the add); then every budget's
    record-boundary prefix of the same validated stream decoded without
    re-encoding into dense bf16 repaired weights, one target set per budget,
    all in one reconstruction pass over the backbone.  Stage
    times come from HIP events on the library's stream; the step time is the
    host wall clock of exactly the timed steps."""
    wl = run.wl
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(STAGES) + 1)]
    acc = dict.fromkeys(STAGES, 0.0)
    bpw_max = max(wl.budgets)
    N = wl.n_weights
    last = run.last

    def step(record: bool):
        ev[0].record(stream)
        for inp, b in zip(run.inputs, run.bb):
            awsrc.awsrc_backbone_rtn(inp["W"], out=b)
        ev[1].record(stream)
        awsrc.awsrc_encode_modules(run.p, run.W_list, run.W0_list, run.d_list, out=run.enc_out, workspace=run.ws)
        ev[2].record(stream)
        s, K, ne = awsrc.awsrc_rank_prefix(run.p, run.shapes, run.mode, bpw_max, run.seed, run.codes, run.scale,
                                           run.gain, workspace=last.get("rws"))
        ev[3].record(stream)
        plan, dws = awsrc.awsrc_decode_prepare(s, [b[3] for b in run.bb], workspace=last.get("dws"))
        ev[4].record(stream)
        awsrc.awsrc_decode_apply(plan)
        ev[5].record(stream)
        prefixes = []
        for bpw in sorted(wl.budgets):
            if run.mode == awsrc.AWSRC_MODE_GLOBAL:
                kb = min(ne, (awsrc.awsrc_budget_bytes(bpw, N) - run.h) // run.L)
            else:
                kb = K
            prefixes.append((bpw, kb))
        # every budget's prefix of the one validated stream, dense bf16, in one pass
        awsrc.awsrc_reconstruct_bf16_prefixes(plan, [kb for _, kb in prefixes], run.outs,
                                              [b[:3] for b in run.bb], 128)
        ev[6].record(stream)
        last.update(K=K, n_eligible=ne, stream_len=int(s.numel()), dws=dws, prefixes=prefixes, plan=plan, s=s)
        if record:
            torch.cuda.synchronize()
            for k, (a, b) in zip(STAGES, zip(ev[:-1], ev[1:])):
                acc[k] += a.elapsed_time(b)

    for _ in range(warmup):
        step(False)
    torch.cuda.synchronize()
    t_wall = 0.0
    for _ in range(steps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        step(True)
        t_wall += time.perf_counter() - t0
    return 1e3 * t_wall / steps, {k: v / steps for k, v in acc.items()}


def encode_roofline(awsrc, run: Run, stage_ms: dict, gen_version: int) -> dict:
    """Roofline of the encoder calls of a step (all of a workload's modules):
    the split matrix-core / vector-ALU bound with the full-score fraction the
    screens report, or the vector-ALU line where no matrix-core screen runs."""
    wl = run.wl
    cand = wl.candidates
    per_elem = wl.d_mode == "elem"
    opc = ops_per_candidate(wl.C, wl.P, per_elem, gen_version)
    enc_s = stage_ms["encode"] / 1e3
    scored = awsrc.awsrc_encode_scored(run.enc_out)
    f_scored = scored / cand
    if mfma_screen(wl.C, wl.P, per_elem, gen_version):
        sb = encode_split_bound(wl.C, wl.P, per_elem, gen_version, f_scored)
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
    extra = {}
    if bound == "alu":
        extra["frac_unpacked_alu"] = achieved / UNPACKED_VALU_TOPS
    return {"bound": bound, "kernel": f"awsrc_encode_modules over the {len(wl.modules)} module(s) of a step "
                                      "(basis, factors, screen, fp64 re-score)",
            "achieved": achieved, "peak": peak, "unit": unit, "frac": achieved / peak, **extra,
            "traffic": measured_traffic("encode", wl.name) if gen_version == 1 else None,
            "traffic_unit": "bytes per step (all encoder calls)", "split": split,
            "ops_per_candidate_unpruned": opc}


def workload_result(awsrc, run: Run, ms_step: float, stage_ms: dict, gen_version: int) -> dict:
    wl = run.wl
    last = run.last
    K = last["K"]
    L = run.L
    dec_bytes = K * (L + 2 * wl.C * 4)  # records, and the fp32 tiles they touch read and written
    t_call = (stage_ms["decode_prepare"] + stage_ms["decode_apply"]) / 1e3
    t_apply = stage_ms["decode_apply"] / 1e3
    dec_gbs = dec_bytes / t_call / 1e9 if t_call > 0 else None
    app_gbs = dec_bytes / t_apply / 1e9 if t_apply > 0 else None
    n_w = wl.n_weights
    n_groups = n_w // 128
    bb_bytes = n_w * (2 if wl.w_dtype == "bf16" else 4) + n_w // 2 + 3 * n_groups + 4 * n_w
    bb_gbs = bb_bytes / (stage_ms["backbone"] / 1e3) / 1e9
    # dense reconstruction of every prefix in one pass: codes 1/2 B per weight
    # and scale and zero 3 B per group read once, bf16 output 2 B per weight
    # and prefix, the longest prefix's records
    n_pref = len(last["prefixes"])
    rc_bytes = n_w // 2 + 3 * n_groups + n_pref * 2 * n_w + max(kb for _, kb in last["prefixes"]) * L
    rc_gbs = rc_bytes / (stage_ms["reconstruct"] / 1e3) / 1e9
    enc_s = stage_ms["encode"] / 1e3
    return {
        "config": {"workload": wl.name, "modules": len(wl.modules), "C": wl.C, "P": wl.P, "b": wl.b, "S": wl.S,
                   "weights": wl.d_mode, "mode": wl.mode, "budgets_bpw": list(wl.budgets), "tiles": wl.n_tiles,
                   "n_weights": n_w, "candidates": wl.candidates, "generator": gen_version},
        "ms_per_step": ms_step,
        "candidates_per_s_step": wl.candidates / (ms_step / 1e3),
        "encode_candidates_per_s": wl.candidates / enc_s,
        "roofline_encode": encode_roofline(awsrc, run, stage_ms, gen_version),
        "decode_add": {"stream_bpw": max(wl.budgets), "records": K, "bytes": dec_bytes,
                       "ms": 1e3 * t_call, "GB/s": dec_gbs,
                       "frac_hbm": dec_gbs / PEAK_HBM_GBS if dec_gbs else None,
                       "apply_ms": 1e3 * t_apply, "apply_GB/s": app_gbs,
                       "apply_frac_hbm": app_gbs / PEAK_HBM_GBS if app_gbs else None,
                       "note": "GB/s and frac_hbm over the whole awsrc_decode_add (validation + apply); "
                               "apply_* for the add alone, as with a prepared plan reused",
                       "traffic": measured_traffic("decode_apply", wl.name)},
        "prefixes": [{"bpw": b, "records": kb} for b, kb in last["prefixes"]],
        "reconstruct_bf16": {"prefixes": len(last["prefixes"]), "bytes": rc_bytes, "ms": stage_ms["reconstruct"],
                             "GB/s": rc_gbs, "frac_hbm": rc_gbs / PEAK_HBM_GBS,
                             "traffic": measured_traffic("reconstruct_bf16", wl.name)},
        "backbone": {"bytes": bb_bytes, "ms": stage_ms["backbone"], "GB/s": bb_gbs,
                     "frac_hbm": bb_gbs / PEAK_HBM_GBS, "traffic": measured_traffic("backbone", wl.name)},
        "stage_ms": stage_ms,
        "stream": {"K": K, "n_eligible": last["n_eligible"], "bytes": last["stream_len"], "L_rec": L},
    }


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=8)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="stack3b")
    ap.add_argument("--extra", default="down3b,block3b,layer32b",
                    help="further workloads timed after the headline one and reported under 'extra' ('' for none)")
    ap.add_argument("--extra-steps", type=int, default=10)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
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
    from synth import workload

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = workload(args.workload)
    log(f"[bench] workload {wl.name}: {len(wl.modules)} module(s), {wl.n_weights} weights, T={wl.n_tiles}, "
        f"S={wl.S}; generating inputs")
    run = Run(awsrc, torch, wl, args.gen_version, dev, sample_step=0 if args.no_cpu_baseline else 256)
    torch.cuda.synchronize()
    log(f"[bench] inputs resident ({torch.cuda.memory_allocated() / 2**30:.1f} GiB); "
        f"{args.warmup} warmup + {args.steps} timed steps")
    ms_step, stage_ms = run_steps(awsrc, torch, run, args.steps, args.warmup)
    res = workload_result(awsrc, run, ms_step, stage_ms, args.gen_version)
    log(f"[bench] {wl.name}: {ms_step:.2f} ms/step, encode {stage_ms['encode']:.2f} ms")
    stream = torch.cuda.current_stream()
    out = {
        "metric": METRIC, "value": wl.candidates / (ms_step / 1e3), "unit": "candidates/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": dict(res["config"], bpw=max(wl.budgets)),
        "roofline": res["roofline_encode"],
        "encode_candidates_per_s": res["encode_candidates_per_s"],
        "decode_add": res["decode_add"],
        "reconstruct_bf16": res["reconstruct_bf16"],
        "backbone": res["backbone"],
        "prefixes": res["prefixes"],
        "stage_ms": stage_ms,
        "stream": res["stream"],
        "device": torch.cuda.get_device_name(0),
    }
    out["backbone_sdq"] = sdq_timing(awsrc, torch, wl, run, stream)
    sample = run.sample
    del run
    torch.cuda.empty_cache()
    extra = {}
    for name in [x for x in args.extra.split(",") if x and x != wl.name]:
        xw = workload(name)
        log(f"[bench] extra workload {name}")
        xr = Run(awsrc, torch, xw, args.gen_version, dev)
        ms_x, st_x = run_steps(awsrc, torch, xr, args.extra_steps, 2)
        extra[name] = workload_result(awsrc, xr, ms_x, st_x, args.gen_version)
        log(f"[bench] {name}: {ms_x:.2f} ms/step, encode {st_x['encode']:.2f} ms")
        del xr
        torch.cuda.empty_cache()
    if extra:
        out["extra"] = extra
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(wl, sample, args.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
