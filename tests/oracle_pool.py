"""Running the oracle's encoder over many tiles for the parity tests.

The oracle is plain fp64 numpy, about a microsecond per (tile, seed); the
full-size parity cases (hundreds of millions of candidates) spread it over
fresh worker processes (`spawn`: nothing of the test process's GPU state is
inherited), one BLAS thread each.  Each worker runs the oracle on its chunk of
tiles with every seed's gain kept and compares the HIP path's outputs for
those tiles against it, so that only a small summary comes back.

Comparison rules (the bars of the encoder parity tests):
* seed: the GPU's seed equals the oracle's, or the oracle's gain for the
  GPU's seed lies within 1e-6 (relative) of the oracle's best gain, plus
  1e-13 of the tile's weighted energy sum_j d_j r_j^2 for gains near zero;
* record: codes and scale field bit-exact for the seed the GPU chose (the
  oracle's record for that seed), unless that candidate has a coefficient
  within 1e-9 of a rounding midpoint or m/qmax within 1e-12 of an fp32
  rounding midpoint (or of a power of two, for power-of-two scales);
* gain within 1e-10 of the tile's energy; unquantized coefficients within
  1e-4 of max |alpha*|.
"""
from __future__ import annotations

import os
import time
from typing import Dict, List, Optional, Sequence

import numpy as np

from oracle import awsrc_oracle as O


def compare_encode(R: np.ndarray, D: np.ndarray, op: "O.Params", g_seed: np.ndarray, g_codes: np.ndarray,
                   g_scale: np.ndarray, g_gain: np.ndarray, g_alpha: Optional[np.ndarray],
                   orc: Optional[Dict[str, np.ndarray]] = None, max_report: int = 8) -> Dict:
    """Check the GPU's per-tile outputs for tiles R, D [N, C] against the
    oracle (run here with every seed's gain unless `orc` is given).  Returns
    counts and the first failures as text."""
    if orc is None:
        orc = O.encode_tiles(R, D, op, keep_all=True)
    N = R.shape[0]
    e = orc["energy"]
    gmax = orc["gain"]
    s_g = g_seed.astype(np.int64)
    s_o = orc["seed"]
    g_at = orc["all_gains"][np.arange(N), s_g]
    fails: List[str] = []

    def bad(mask, what):
        for i in np.flatnonzero(mask)[: max(0, max_report - len(fails))]:
            fails.append(f"tile {i}: {what}")
        return int(np.count_nonzero(mask))

    n_fail = bad(~(np.abs(g_at - gmax) <= 1e-6 * np.abs(gmax) + 1e-13 * e), "seed outside the tie window")
    same = s_g == s_o
    flagged = orc["flag_half"] | orc["flag_scale"]
    exact = same & ~flagged
    n_fail += bad(exact & np.any(g_codes != orc["codes"], axis=1), "codes differ")
    n_fail += bad(exact & (g_scale != orc["scale"]), "scale differs")
    n_fail += bad(same & ~(np.abs(g_gain - gmax) <= 1e-10 * e + 1e-300), "gain differs")
    if g_alpha is not None:
        amax = np.abs(orc["alpha"]).max(axis=1)
        n_fail += bad(same & ~(np.abs(g_alpha - orc["alpha"]).max(axis=1) <= 1e-4 * amax + 1e-30),
                      "alpha differs")
    n_edge = int(np.count_nonzero(same & flagged))
    diff = np.flatnonzero(~same)
    for i in diff:
        q, bits, g, alpha = O.candidate(R[i], D[i], op, int(s_g[i]))
        ok = abs(g_gain[i] - g) <= 1e-10 * e[i] + 1e-300
        qm, _, sc = O.quantize(alpha[None], op.b, op.scale_fmt)
        edge = bool(O._boundary_flags(alpha[None], sc, op.qmax)[0]
                    or O._scale_flags(alpha[None], op.qmax, scale_fmt=op.scale_fmt)[0])
        n_edge += int(edge)
        if not edge:
            ok = ok and np.array_equal(g_codes[i], q) and int(g_scale[i]) == bits
        if g_alpha is not None:
            ok = ok and np.abs(g_alpha[i] - alpha).max() <= 1e-4 * np.abs(alpha).max() + 1e-30
        if not ok:
            n_fail += 1
            if len(fails) < max_report:
                fails.append(f"tile {i}: record of tied seed {int(s_g[i])} differs from the oracle's")
    return {"tiles": N, "seed_diff": int(diff.size), "edge": n_edge, "failures": n_fail, "report": fails}


def _job(args):
    """Worker: the oracle on one chunk and the comparison; one BLAS thread."""
    from threadpoolctl import threadpool_limits

    (tag, R, D, op, g_seed, g_codes, g_scale, g_gain, g_alpha) = args
    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
        out = compare_encode(R, D, op, g_seed, g_codes, g_scale, g_gain, g_alpha)
    out["seconds"] = time.perf_counter() - t0
    out["tag"] = tag
    out["report"] = [f"{tag} {r}" for r in out["report"]]
    return out


def n_workers() -> int:
    # the host's CPU share per GPU is 16 cores, whatever the affinity mask shows
    return max(1, min(16, len(os.sched_getaffinity(0))))


def chunk_jobs(tag: str, R, D, op, g_seed, g_codes, g_scale, g_gain, g_alpha, n_chunks: int) -> List[tuple]:
    """Cut one tile set into contiguous chunks (tiles keep their order)."""
    N = R.shape[0]
    step = max(1, -(-N // max(1, n_chunks)))
    jobs = []
    for i in range(0, N, step):
        sl = slice(i, min(N, i + step))
        jobs.append((f"{tag}[{i}:{sl.stop}]", R[sl], D[sl], op, g_seed[sl], g_codes[sl], g_scale[sl], g_gain[sl],
                     None if g_alpha is None else g_alpha[sl]))
    return jobs


def run_jobs(jobs: Sequence[tuple], nproc: Optional[int] = None) -> Dict:
    """Run the comparison jobs over a spawn pool and sum their summaries."""
    import multiprocessing as mp

    nproc = nproc or n_workers()
    t0 = time.perf_counter()
    if nproc == 1 or len(jobs) == 1:
        outs = [_job(j) for j in jobs]
    else:
        outs = []
        with mp.get_context("spawn").Pool(min(nproc, len(jobs))) as pool:
            # a line per finished chunk, so that a long comparison shows its progress
            for o in pool.imap_unordered(_job, jobs, chunksize=1):
                outs.append(o)
                print(f"[oracle_pool] {len(outs)}/{len(jobs)} chunks, {time.perf_counter() - t0:.1f} s", flush=True)
    tot = {"tiles": 0, "seed_diff": 0, "edge": 0, "failures": 0, "report": [], "cpu_seconds": 0.0}
    for o in outs:
        for k in ("tiles", "seed_diff", "edge", "failures"):
            tot[k] += o[k]
        tot["cpu_seconds"] += o["seconds"]
        tot["report"].extend(o["report"])
    tot["wall_seconds"] = time.perf_counter() - t0
    tot["workers"] = nproc
    return tot
