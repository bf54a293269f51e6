"""CPU checks of the comparison the full-size GPU parity tests run
(tests/oracle_pool.py): the oracle's own records pass, a tied seed with its
own record passes, and altered records, out-of-window seeds, gains and
coefficients fail; the spawn pool sums what its workers report."""
import numpy as np

import oracle_pool as OP
from oracle import awsrc_oracle as O


def _case(n=40, seed=1):
    rng = np.random.default_rng(seed)
    op = O.Params(C=16, P=4, b=4, S=16, basis_key=5, ridge_lambda=1e-6)
    R = rng.normal(0, 0.01, (n, 16))
    D = np.exp(rng.normal(0, 1.5, (n, 16)))
    orc = O.encode_tiles(R, D, op, keep_all=True)
    g = {"g_seed": orc["seed"].copy(), "g_codes": orc["codes"].copy(), "g_scale": orc["scale"].copy(),
         "g_gain": orc["gain"].copy(), "g_alpha": orc["alpha"].astype(np.float32)}
    return op, R, D, orc, g


def test_oracle_records_pass():
    op, R, D, orc, g = _case()
    out = OP.compare_encode(R, D, op, **g, orc=orc)
    assert out["failures"] == 0 and out["seed_diff"] == 0 and out["tiles"] == 40


def test_tied_seed_with_its_own_record_passes():
    # a tile whose gain is the same for two seeds: zero residual except one
    # coordinate is not enough; instead duplicate a seed's basis by giving the
    # tile a residual in the span shared by every basis (all-zero residual)
    op, R, D, orc, g = _case()
    R[3] = 0.0
    orc = O.encode_tiles(R, D, op, keep_all=True)
    g = {"g_seed": orc["seed"].copy(), "g_codes": orc["codes"].copy(), "g_scale": orc["scale"].copy(),
         "g_gain": orc["gain"].copy(), "g_alpha": orc["alpha"].astype(np.float32)}
    g["g_seed"][3] = 7            # every seed ties at gain 0
    out = OP.compare_encode(R, D, op, **g, orc=orc)
    assert out["failures"] == 0 and out["seed_diff"] == 1


def test_altered_records_fail():
    op, R, D, orc, g0 = _case()
    worst = int(np.argmin(orc["all_gains"][0]))
    cases = {
        "codes": lambda g: g["g_codes"].__setitem__((5, 0), g["g_codes"][5, 0] + 1),
        "scale": lambda g: g["g_scale"].__setitem__(6, g["g_scale"][6] + 1),
        "gain": lambda g: g["g_gain"].__setitem__(7, g["g_gain"][7] * (1 + 1e-6)),
        "alpha": lambda g: g["g_alpha"].__setitem__((8, 1), g["g_alpha"][8, 1] + 1e-3 * abs(g["g_alpha"][8]).max()),
        "seed": lambda g: g["g_seed"].__setitem__(0, worst),
    }
    for name, f in cases.items():
        g = {k: v.copy() for k, v in g0.items()}
        f(g)
        out = OP.compare_encode(R, D, op, **g, orc=orc)
        assert out["failures"] >= 1, name


def test_pool_sums_worker_summaries():
    op, R, D, orc, g = _case(n=64, seed=3)
    g["g_codes"][50, 2] += 1
    jobs = OP.chunk_jobs("t", R, D, op, g["g_seed"], g["g_codes"], g["g_scale"], g["g_gain"], g["g_alpha"], 4)
    assert len(jobs) == 4 and sum(j[1].shape[0] for j in jobs) == 64
    tot = OP.run_jobs(jobs, nproc=2)
    assert tot["tiles"] == 64 and tot["failures"] == 1
    assert any("t[48:64] tile 2" in r for r in tot["report"])
