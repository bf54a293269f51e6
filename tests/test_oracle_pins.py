"""Pins of the CPU oracle against facts that do not come from the oracle itself:
published generator outputs, printed byte counts, closed forms, textbook
reductions, invariants and brute force on tiny inputs."""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest

from conftest import read_golden, read_golden_lines
from oracle import awsrc_oracle as O


# ---------------------------------------------------------------- generator
def test_splitmix64_published_vectors():
    want = [int(x, 16) for x in read_golden_lines("splitmix64_key0.txt")]
    assert [O.splitmix64(0, n) for n in range(len(want))] == want


def _splitmix64_numpy(key, counters):
    """Independent numpy uint64 implementation (wrapping arithmetic)."""
    with np.errstate(over="ignore"):
        z = np.uint64(key) + (counters.astype(np.uint64) + np.uint64(1)) * np.uint64(0x9E3779B97F4A7C15)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        return z ^ (z >> np.uint64(31))


@pytest.mark.parametrize("key", [0, 1, 0xDEADBEEFCAFEF00D, (1 << 64) - 1])
def test_splitmix64_two_implementations(key):
    rng = np.random.default_rng(key & 0xFFFF)
    n = np.concatenate([np.arange(2000), rng.integers(0, 1 << 62, 2000)]).astype(np.uint64)
    got = _splitmix64_numpy(key, n)
    for i in range(0, len(n), 97):
        assert int(got[i]) == O.splitmix64(key, int(n[i]))


def test_gen_basis_worked_example():
    g = read_golden("gen_v1_key0_s0_C64_P4.txt")
    word = int(g["sign_word"][0], 16)
    sigma, cols = O.gen_basis(0, 0, 64, 4)
    assert cols == [int(c) for c in g["columns"]]
    assert all(sigma[j] == (-1 if (word >> j) & 1 else 1) for j in range(64))


@pytest.mark.parametrize("C,P", [(4, 2), (16, 4), (64, 8), (128, 8), (64, 64), (32, 1)])
def test_gen_basis_properties(C, P):
    for s in range(40):
        sigma, cols = O.gen_basis(7, s, C, P)
        assert len(cols) == P and len(set(cols)) == P
        assert all(0 <= c < C for c in cols)
        assert set(np.unique(sigma)) <= {-1, 1}
    # signs of C=128 use two words; the second half must differ from the first
    if C == 128:
        sig, _ = O.gen_basis(0, 3, 128, 1)
        w0, w1 = O.basis_word(0, 3, 0), O.basis_word(0, 3, 1)
        assert all(sig[64 + j] == (-1 if (w1 >> j) & 1 else 1) for j in range(64))
        assert all(sig[j] == (-1 if (w0 >> j) & 1 else 1) for j in range(64))


def test_gen_basis_full_selection_is_permutation():
    # P = C draws every column exactly once
    for s in range(10):
        _, cols = O.gen_basis(3, s, 16, 16)
        assert sorted(cols) == list(range(16))


# ---------------------------------------------------------------- generator version 2
def test_gen_v2_worked_example():
    g = read_golden("gen_v2_key0_s0_C4_P1.txt")
    sigma, cols = O.gen_basis(0, 0, 4, 1)
    assert [int(x) for x in g["sigma"]] == list(sigma) and cols == [int(c) for c in g["columns"]]
    assert list(O.gen_permutation(0, 0, 4, 1)) == [int(x) for x in g["perm"]]
    B = O.basis_matrix(0, 0, 4, 1, gen_version=2)
    assert np.array_equal(B[:, 0] * 2, np.array([int(x) for x in g["basis_col0_times2"]], dtype=float))


@pytest.mark.parametrize("C,P", [(4, 2), (16, 4), (64, 8), (128, 8), (128, 16)])
def test_gen_v2_is_v1_with_permuted_hadamard_rows(C, P):
    """Signs and columns are version 1's words; the permutation is a bijection
    of the coordinates; B[j, p] sigma_j sqrt(C) = H[pi(j), c_p]; columns stay
    orthonormal."""
    H = O.hadamard(C)
    for s in range(12):
        sigma, cols = O.gen_basis(11, s, C, P)
        pi = O.gen_permutation(11, s, C, P)
        assert sorted(pi) == list(range(C))
        B2 = O.basis_matrix(11, s, C, P, gen_version=2)
        B1 = O.basis_matrix(11, s, C, P, gen_version=1)
        assert np.array_equal(B1 * math.sqrt(C) * sigma[:, None], H[:, cols].astype(float))
        assert np.allclose(B2 * math.sqrt(C) * sigma[:, None], H[pi][:, cols], atol=1e-12)
        assert np.allclose(B2.T @ B2, np.eye(P), atol=1e-12)


def test_gen_v2_permutation_uniform_and_independent_of_the_columns():
    """C = 4, P = 1: over 48,000 seeds every one of the 24 permutations is
    equally likely, and the permutation is independent of the column draw
    (chi-square at p = 1e-6); a shuffle that reused or overlapped the column
    and sign words, or a biased shuffle, fails one of these."""
    from scipy.stats import chi2
    perms = {p: i for i, p in enumerate(itertools.permutations(range(4)))}
    n = 48000
    joint = np.zeros((4, 24))
    for s in range(n):
        _, cols = O.gen_basis(5, s, 4, 1)
        joint[cols[0], perms[tuple(O.gen_permutation(5, s, 4, 1))]] += 1
    marg = joint.sum(axis=0)
    x2 = float(np.sum((marg - n / 24) ** 2 / (n / 24)))
    assert x2 < chi2.ppf(1 - 1e-6, 23)
    expect = np.outer(joint.sum(axis=1), marg) / n
    x2j = float(np.sum((joint - expect) ** 2 / expect))
    assert x2j < chi2.ppf(1 - 1e-6, 3 * 23)


# ---------------------------------------------------------------- Hadamard
@pytest.mark.parametrize("C", [1, 2, 4, 8, 16, 32, 64, 128])
def test_hadamard_orthogonal(C):
    H = O.hadamard(C)
    assert np.array_equal(H @ H.T, C * np.eye(C, dtype=np.int64))


def test_hadamard_sylvester_recursion():
    H = np.array([[1]], dtype=np.int64)
    for k in range(7):
        H = np.block([[H, H], [H, -H]])
        assert np.array_equal(H, O.hadamard(2 ** (k + 1)))


def test_basis_columns_orthonormal():
    B = O.basis_matrix(0, 5, 64, 8)
    assert np.allclose(B.T @ B, np.eye(8), atol=1e-15)


# ---------------------------------------------------------------- backbone
def test_rtn_closed_form_group():
    # w_k = (k mod 16)/4 - 1: min -1, max 2.75, (max-min)/15 = 0.25 exactly,
    # zero point rint(1/0.25) = 4, codes k mod 16, reconstruction exact.
    k = np.arange(128)
    W = ((k % 16) * 0.25 - 1.0).astype(np.float32)[None, :]
    codes, scale, zero, W0 = O.rtn_backbone(W)
    assert scale[0, 0] == 0x3400 and zero[0, 0] == 4
    q = np.empty(128, np.int64)
    q[0::2] = codes[0] & 15
    q[1::2] = codes[0] >> 4
    assert np.array_equal(q, k % 16)
    assert np.array_equal(W0, W)


def test_rtn_half_even_tie():
    # scale 1.0 (max-min = 15), zero point 0; w = 2.5 -> rint -> 2, w = 3.5 -> 4
    W = np.zeros((1, 128), np.float32)
    W[0, 1] = 15.0
    W[0, 2] = 2.5
    W[0, 3] = 3.5
    codes, scale, zero, W0 = O.rtn_backbone(W)
    assert scale[0, 0] == 0x3C00 and zero[0, 0] == 0
    assert W0[0, 2] == 2.0 and W0[0, 3] == 4.0 and W0[0, 1] == 15.0


def test_rtn_degenerate_group():
    W = np.full((1, 128), 0.5, np.float32)
    codes, scale, zero, W0 = O.rtn_backbone(W)
    assert scale[0, 0] == 0x3C00 and zero[0, 0] == 0 and np.all(codes == 0) and np.all(W0 == 0)


def test_rtn_nearest_code_exact_rational():
    """Every code is a nearest integer of w/s + z, checked in exact rational
    arithmetic (independent of float rounding except at exact ties)."""
    rng = np.random.default_rng(0)
    W = (rng.standard_normal((8, 256)) * 0.02).astype(np.float32)
    W[3, :128] *= 100
    codes, scale, zero, W0 = O.rtn_backbone(W)
    for r in range(8):
        for g in range(2):
            s = Fraction(float(np.array([scale[r, g]], np.uint16).view(np.float16)[0]))
            z = int(zero[r, g])
            grp = W[r, g * 128:(g + 1) * 128]
            mn, mx = Fraction(float(grp.min())), Fraction(float(grp.max()))
            # the stored scale is the fp16 rounding of (max-min)/15 within fp16/fp32 error
            assert abs(s - (mx - mn) / 15) <= (mx - mn) / 15 * Fraction(1, 1024)
            assert 0 <= z <= 15 and abs(Fraction(z) - (-mn / s)) <= Fraction(1, 2) + Fraction(1, 10 ** 6)
            for i in range(128):
                col = g * 128 + i
                q = int((codes[r, col // 2] >> (4 * (col % 2))) & 15)
                x = Fraction(float(grp[i])) / s + z
                if 0 < q < 15:
                    assert abs(x - q) <= Fraction(1, 2) + Fraction(1, 10 ** 6)
                elif q == 0:
                    assert x <= Fraction(1, 2) + Fraction(1, 10 ** 6)
                else:
                    assert x >= Fraction(29, 2) - Fraction(1, 10 ** 6)
                assert float(W0[r, col]) == float((q - z) * s)


# ---------------------------------------------------------------- fit
def _random_problem(rng, N, C, per_element=True):
    R = rng.standard_normal((N, C)) * 0.01
    D = np.exp(rng.standard_normal((N, C)) * 1.5) if per_element else np.tile(
        np.exp(rng.standard_normal(C) * 1.5), (N, 1))
    return R, D


@pytest.mark.parametrize("lam", [0.0, 1e-6, 0.3])
def test_fit_matches_lstsq(lam):
    """Eq. (3) is the least-squares problem [D^1/2 B; sqrt(eps) I] a ~ [D^1/2 r; 0]."""
    rng = np.random.default_rng(1)
    R, D = _random_problem(rng, 20, 64)
    B = O.basis_matrix(0, 9, 64, 8)
    alpha, G, b = O.fit(R, D, B, lam)
    for t in range(20):
        eps = lam * D[t].mean()
        A = np.vstack([np.sqrt(D[t])[:, None] * B, math.sqrt(eps) * np.eye(8)])
        y = np.concatenate([np.sqrt(D[t]) * R[t], np.zeros(8)])
        ref = np.linalg.lstsq(A, y, rcond=None)[0]
        assert np.allclose(alpha[t], ref, rtol=1e-10, atol=1e-14 * np.abs(ref).max())


def test_fit_first_order_optimality():
    """The objective of Eq. (3) does not decrease along any coordinate direction."""
    rng = np.random.default_rng(2)
    R, D = _random_problem(rng, 5, 32)
    B = O.basis_matrix(1, 2, 32, 4)
    lam = 1e-3
    alpha, _, _ = O.fit(R, D, B, lam)

    def obj(t, a):
        return float(np.sum(D[t] * (B @ a - R[t]) ** 2) + lam * D[t].mean() * np.sum(a * a))

    for t in range(5):
        f0 = obj(t, alpha[t])
        for p in range(4):
            for h in (1e-5, -1e-5):
                e = np.zeros(4)
                e[p] = h * max(1e-3, abs(alpha[t][p]))
                assert obj(t, alpha[t] + e) >= f0 - 1e-18


def test_gram_and_projection_via_walsh_hadamard():
    """G_pq = WHT(d)[c_p xor c_q]/C and b_p = WHT(sigma*d*r)[c_p]/sqrt(C)
    (sign cancellation and the Sylvester xor identity H[j,a]H[j,b] = H[j,a^b])."""

    def fwht(v):  # fast Walsh-Hadamard transform, natural order
        v = v.astype(np.float64).copy()
        h = 1
        while h < len(v):
            for i in range(0, len(v), 2 * h):
                a, b = v[i:i + h].copy(), v[i + h:i + 2 * h].copy()
                v[i:i + h], v[i + h:i + 2 * h] = a + b, a - b
            h *= 2
        return v

    rng = np.random.default_rng(3)
    C, P = 64, 8
    R, D = _random_problem(rng, 6, C)
    for s in range(4):
        sigma, cols = O.gen_basis(0, s, C, P)
        B = O.basis_matrix(0, s, C, P)
        _, G, b = O.fit(R, D, B, 0.0)
        for t in range(6):
            wd = fwht(D[t])
            Gx = np.array([[wd[cp ^ cq] / C for cq in cols] for cp in cols])
            assert np.allclose(G[t], Gx, rtol=1e-12, atol=1e-15)
            wu = fwht(sigma * D[t] * R[t])
            assert np.allclose(b[t], wu[cols] / math.sqrt(C), rtol=1e-12, atol=1e-16)
            assert np.isclose(G[t][0, 0], D[t].mean(), rtol=1e-13)


# ---------------------------------------------------------------- quantize / score
def test_gain_coefficient_space_identity():
    """sum_j d(r^2 - (r - B a)^2) = 2 a^T b - a^T (B^T D B) a for any a."""
    rng = np.random.default_rng(4)
    R, D = _random_problem(rng, 30, 64)
    B = O.basis_matrix(0, 3, 64, 8)
    alpha, G, b = O.fit(R, D, B, 1e-6)
    q, bits, sc = O.quantize(alpha, 4)
    ah = sc[:, None] * q
    g_def = O.weighted_gain(R, D, ah @ B.T)
    G0 = G - (1e-6 * D.mean(axis=1))[:, None, None] * np.eye(8)
    g_cs = 2 * np.einsum("np,np->n", ah, b) - np.einsum("np,npq,nq->n", ah, G0, ah)
    assert np.allclose(g_def, g_cs, rtol=1e-11, atol=1e-20)


def test_quantize_properties():
    rng = np.random.default_rng(5)
    alpha = rng.standard_normal((500, 8)) * 0.05
    alpha[0] = 0
    for b in (2, 3, 4, 8):
        qmax = 2 ** (b - 1) - 1
        q, bits, sc = O.quantize(alpha, b)
        assert np.all(np.abs(q) <= qmax)
        assert np.all(np.abs(q[1:]).max(axis=1) == qmax)
        assert bits[0] == 0 and np.all(q[0] == 0)
        # scale is fp16(fp32(m/qmax)): within half an fp16 ulp (plus fp32 rounding) of m/qmax
        m = np.abs(alpha[1:]).max(axis=1)
        assert np.all(np.abs(sc[1:] - m / qmax) <= (m / qmax) * (2.0 ** -11 + 2.0 ** -24))
        # each code is a nearest integer of alpha/scale
        x = alpha[1:] / sc[1:, None]
        assert np.all(np.abs(x - q[1:]) <= 0.5 + 1e-12)


def test_quantize_fp16_double_rounding():
    """The scale rounds m/qmax to fp32 first, then to fp16 (both to nearest even)."""
    # v sits just above an fp16 midpoint in float64 but rounds onto it in fp32:
    # 1 + 2^-11 is the fp16 midpoint between 1 and 1+2^-10; fp32 of 1 + 2^-11 + 2^-40
    # is exactly the midpoint, which then ties to even (1.0); direct rounding gives 1+2^-10.
    v = 1 + 2.0 ** -11 + 2.0 ** -40
    q, bits, sc = O.quantize(np.array([[7 * v, 0.0]]), 4)
    assert bits[0] == 0x3C00
    assert np.float16(v) != np.float16(1.0)  # the direct rounding would differ


def test_quantize_saturates_fp16():
    q, bits, sc = O.quantize(np.array([[1e6, -3e5]]), 4)
    assert bits[0] == 0x7BFF and q[0, 0] == 7


# ---------------------------------------------------------------- exact cases
def test_exact_reconstruction_full_basis():
    """P = C, unit weights, eps = 0, unquantized: every seed reproduces r exactly."""
    rng = np.random.default_rng(6)
    C = 16
    R = rng.standard_normal((12, C))
    D = np.ones((12, C))
    p = O.Params(C=C, P=C, b=4, S=6, ridge_lambda=0.0)
    enc = O.encode_tiles(R, D, p, quantize_coeffs=False, keep_all=True)
    energy = np.sum(R * R, axis=1)
    assert np.allclose(enc["all_gains"], energy[:, None], rtol=1e-12)
    for t in range(12):
        B = O.basis_matrix(0, int(enc["seed"][t]), C, C)
        assert np.allclose(B @ enc["alpha"][t], R[t], atol=1e-12)


def test_orthonormal_basis_quantized_parseval():
    """P = C, unit weights, eps = 0: alpha* = B^T r, and the quantized gain is
    |r|^2 - |alpha* - alpha_hat|^2 (Parseval for an orthonormal basis)."""
    rng = np.random.default_rng(7)
    C = 16
    R = rng.standard_normal((40, C)) * 0.1
    D = np.ones((40, C))
    p = O.Params(C=C, P=C, b=3, S=5, ridge_lambda=0.0)
    enc = O.encode_tiles(R, D, p, keep_all=True)
    for s in range(5):
        B = O.basis_matrix(0, s, C, C)
        a_star = R @ B
        q, bits, sc = O.quantize(a_star, 3)
        want = np.sum(R * R, axis=1) - np.sum((a_star - sc[:, None] * q) ** 2, axis=1)
        assert np.allclose(enc["all_gains"][:, s], want, rtol=1e-11, atol=1e-15)


def test_ls_bound_and_zero_tile():
    """eps = 0: no quantized reconstruction beats the least-squares optimum b^T G^-1 b;
    an all-zero tile gives gain 0 for every seed and keeps seed 0 (lowest wins ties)."""
    rng = np.random.default_rng(8)
    R, D = _random_problem(rng, 64, 64)
    R[5] = 0
    p = O.Params(C=64, P=8, b=4, S=16, ridge_lambda=0.0)
    enc = O.encode_tiles(R, D, p, keep_all=True)
    for s in range(16):
        B = O.basis_matrix(0, s, 64, 8)
        alpha, G, b = O.fit(R, D, B, 0.0)
        bound = np.einsum("np,np->n", alpha, b)
        assert np.all(enc["all_gains"][:, s] <= bound * (1 + 1e-12) + 1e-30)
    assert enc["seed"][5] == 0 and enc["gain"][5] == 0 and enc["scale"][5] == 0
    assert np.all(enc["codes"][5] == 0)


def test_tie_keeps_lowest_seed():
    rng = np.random.default_rng(9)
    R, D = _random_problem(rng, 10, 16)
    B0 = O.basis_matrix(0, 0, 16, 2)
    B1 = O.basis_matrix(0, 1, 16, 2)
    enc = O.encode_tiles(R, D, O.Params(C=16, P=2, b=4, S=3), bases=[B1, B0, B1])
    assert np.all(np.isin(enc["seed"], [0, 1]))


# ---------------------------------------------------------------- brute force
def _solve_small(G, b):
    """Cramer's rule in plain Python for P <= 2."""
    if len(b) == 1:
        return [b[0] / G[0][0]]
    det = G[0][0] * G[1][1] - G[0][1] * G[1][0]
    return [(b[0] * G[1][1] - G[0][1] * b[1]) / det, (G[0][0] * b[1] - b[0] * G[1][0]) / det]


def _brute_error(r, d, sigma, cols, lam, b):
    C = len(r)
    P = len(cols)
    col = [[sigma[j] * (-1 if bin(j & c).count("1") % 2 else 1) / math.sqrt(C) for j in range(C)]
           for c in cols]
    eps = lam * sum(d) / C
    G = [[sum(d[j] * col[p][j] * col[q][j] for j in range(C)) + (eps if p == q else 0.0)
          for q in range(P)] for p in range(P)]
    bb = [sum(d[j] * col[p][j] * r[j] for j in range(C)) for p in range(P)]
    a = _solve_small(G, bb)
    qmax = 2 ** (b - 1) - 1
    m = max(abs(x) for x in a)
    sc = float(np.float16(np.float32(m / qmax)))
    q = [max(-qmax, min(qmax, round(x / sc))) for x in a] if sc > 0 else [0] * P
    rhat = [sum(sc * q[p] * col[p][j] for p in range(P)) for j in range(C)]
    return sum(d[j] * (r[j] - rhat[j]) ** 2 for j in range(C))


@pytest.mark.parametrize("C,P", [(4, 1), (4, 2), (8, 2)])
def test_brute_force_selection(C, P):
    """Over an exhaustive basis set (every sign pattern x every ordered column
    choice) the oracle's choice attains the minimum weighted error after
    rounding, computed independently in plain Python."""
    rng = np.random.default_rng(10 + C + P)
    H = O.hadamard(C)
    signs = list(itertools.product([1, -1], repeat=C))
    if C == 8:
        signs = signs[::5]
    colsets = list(itertools.permutations(range(C), P))
    combos = [(np.array(sg), list(cs)) for sg in signs for cs in colsets]
    bases = [(sg[:, None] * H[:, cs]).astype(np.float64) / math.sqrt(C) for sg, cs in combos]
    R, D = _random_problem(rng, 6, C)
    lam = 1e-6
    enc = O.encode_tiles(R, D, O.Params(C=C, P=P, b=3, S=len(bases), ridge_lambda=lam), bases=bases)
    for t in range(6):
        errs = [_brute_error(list(R[t]), list(D[t]), sg, cs, lam, 3) for sg, cs in combos]
        best = min(errs)
        chosen = errs[int(enc["seed"][t])]
        energy = float(np.sum(D[t] * R[t] ** 2))
        assert chosen <= best + 1e-12 * energy
        assert abs((energy - chosen) - enc["gain"][t]) <= 1e-10 * energy


# ---------------------------------------------------------------- accounting
def test_paper_byte_accounting():
    g = read_golden("paper_accounting.txt")
    L, h, K = int(g["record_bytes"][0]), int(g["header_bytes"][0]), int(g["K"][0])
    n_mod, N = int(g["n_modules"][0]), int(g["n_scope"][0])
    C, P, b, S = (int(g[k][0]) for k in "CPbS")
    assert h + L * K == int(g["sidecar_bytes"][0])
    assert round(8 * (h + L * K) / N, 3) == float(g["delta_scope_bpw"][0])
    T = N // C
    p = O.Params(C=C, P=P, b=b, S=S, idx_bits=0)
    assert O.index_bits(p, T) == 28
    for b_e in range(1, 9):
        assert O.record_bytes(p, T, scale_bits=b_e) == L
    assert O.record_bytes(p, T, scale_bits=9) == L + 1
    assert O.header_bytes(n_mod) == h
    # the 4.23-bpw prefix: K records fit a budget of h + L*K bytes
    assert O.prefix_K(h + L * K, h, L, 10 ** 9) == K
    assert O.prefix_K(h + L * K + L - 1, h, L, 10 ** 9) == K


def test_small_config_record_size():
    # 32-bit index + 6-bit seed + 4x4-bit codes + 16-bit scale = 70 bits -> 9 bytes
    assert O.record_bytes(O.Params(C=64, P=4, b=4, S=64), 1024) == 9
    assert O.record_bytes(O.Params(C=64, P=8, b=4, S=256), 352256) == 11
    assert O.record_bytes(O.Params(C=128, P=8, b=3, S=1024), 3809280) == 11
    assert O.record_bytes(O.Params(C=64, P=8, b=4, S=512), 43352064) == 12


def test_prefix_K_rules():
    assert O.prefix_K(1327, 48, 9, 1000) == (1327 - 48) // 9
    assert O.prefix_K(1327, 48, 9, 3) == 3
    with pytest.raises(ValueError):
        O.prefix_K(47, 48, 9, 10)
    assert O.budget_bytes(0.162, 65536) == 1327


# ---------------------------------------------------------------- records / stream
def test_record_worked_example():
    g = read_golden("rec_v1_example.txt")
    rec = O.pack_record(int(g["idx"][0]), int(g["seed"][0]), [int(c) for c in g["codes"]],
                        int(g["scale"][0], 16), 32, 6, 4, 9)
    assert rec == bytes(int(x, 16) for x in g["bytes"])
    assert O.unpack_record(rec, 32, 6, 4, 4) == (int(g["idx"][0]), 5, [1, -1, 7, -7], 0x3C00)


@pytest.mark.parametrize("ib,S,P,b", [(32, 64, 4, 4), (28, 16, 4, 4), (32, 1024, 8, 3), (20, 65536, 16, 8),
                                      (32, 2, 1, 2)])
def test_record_round_trip_extremes(ib, S, P, b):
    sb = O.seed_bits(S)
    L = (ib + sb + P * b + 16 + 7) // 8
    qmax = 2 ** (b - 1) - 1
    for idx in (0, (1 << ib) - 1, 12345 % (1 << ib)):
        for seed in (0, S - 1):
            for codes in ([qmax] * P, [-qmax] * P, [(-1) ** i * (i % (qmax + 1)) for i in range(P)]):
                for sc in (0x0001, 0x7BFF, 0x3C00, 0x0000):
                    rec = O.pack_record(idx, seed, codes, sc, ib, sb, b, L)
                    assert len(rec) == L
                    assert O.unpack_record(rec, ib, sb, P, b) == (idx, seed, codes, sc)


def test_stream_header_layout():
    p = O.Params(C=16, P=4, b=4, S=16, basis_key=0x0123456789ABCDEF, idx_bits=0)
    mods = [(2048, 11008)] * 108
    hdr = O.stream_header(p, mods, per_module=False)
    assert len(hdr) == 904
    hd = O.parse_header(hdr)
    # 28-bit index + 4-bit seed + 16 code bits + 16-bit fp16 scale = 64 bits; the
    # paper's 7-byte record needs a scale exponent of at most 8 bits instead
    assert hd["T_total"] == 108 * 2048 * 11008 // 16 and hd["L_rec"] == 8 and hd["basis_key"] == p.basis_key
    assert hd["idx_bits"] == 28 and hd["seed_bits"] == 4 and hd["modules"][107] == (2048, 11008)


def test_rank_order_ties_and_eligibility():
    gain = np.array([0.5, 2.0, -1.0, 2.0, 0.0, 0.5, 3.0])
    order = O.rank_order(gain, np.arange(7))
    assert list(order) == [6, 1, 3, 0, 5]


# ---------------------------------------------------------------- end to end
def _small_module(seed=0, rows=8, cols=256, d_col=True):
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((rows, cols)) * 0.02).astype(np.float32)
    d = np.exp(rng.standard_normal(cols)) if d_col else np.exp(rng.standard_normal((rows, cols)))
    return W, d


def _encode_module(W, d, p):
    codes, scale, zero, W0 = O.rtn_backbone(W)
    R = O.residual(W, W0)
    rows, cols = W.shape
    enc = O.encode_tiles(O.tiles(R, p.C), O.tile_weights(d, rows, cols, p.C), p)
    return W0, enc


@pytest.mark.parametrize("gen_version", [1, 2])
def test_prefix_decodability_every_prefix(gen_version):
    """Every record-boundary prefix decodes against the same W0: the weighted
    error drops by exactly the listed gains, and the empty prefix is W0 itself
    (the decoder regenerates the bases of the generator the header names)."""
    W, d = _small_module()
    p = O.Params(C=64, P=4, b=4, S=16, gen_version=gen_version)
    W0, enc = _encode_module(W, d, p)
    stream, K, n_elig = O.build_stream(p, [W.shape], enc, bpw=8.0, per_module=False)
    h = O.header_bytes(1)
    L = O.record_bytes(p, enc["gain"].size)
    assert K == n_elig and len(stream) == h + K * L
    order = O.rank_order(enc["gain"], np.arange(enc["gain"].size))
    e0 = O.weighted_error(W, W0.astype(np.float64), d)
    prev = e0
    for k in range(K + 1):
        (What,) = O.decode_add(stream[:h + k * L], [W0])
        if k == 0:
            assert np.array_equal(What, W0.astype(np.float64))
        e = O.weighted_error(W, What, d)
        want = e0 - float(np.sum(enc["gain"][order[:k]]))
        assert abs(e - want) <= 1e-9 * e0
        assert e <= prev * (1 + 1e-12)
        prev = e


def test_per_module_quota_and_determinism():
    p = O.Params(C=64, P=4, b=4, S=8)
    mods, encs = [], []
    for s in range(3):
        W, d = _small_module(seed=s, rows=4 + 4 * s)
        W0, enc = _encode_module(W, d, p)
        mods.append(W.shape)
        encs.append(enc)
    cat = {k: np.concatenate([e[k] for e in encs]) for k in ("seed", "codes", "scale", "gain")}
    s1, K, _ = O.build_stream(p, mods, cat, bpw=0.5, per_module=True)
    s2, K2, _ = O.build_stream(p, mods, cat, bpw=0.5, per_module=True)
    assert s1 == s2 and K == K2
    L = O.record_bytes(p, sum(r * c // 64 for r, c in mods))
    want = sum(min(int(np.sum(e["gain"] > 0)), O.budget_bytes(0.5, r * c) // L) for e, (r, c) in zip(encs, mods))
    assert K == want and len(s1) == O.header_bytes(3) + K * L
    # sections follow module order
    hd = O.parse_header(s1)
    idx = [O.unpack_record(s1[hd["h"] + i * L: hd["h"] + (i + 1) * L], 32, 3, 4, 4)[0] for i in range(K)]
    mod_of = np.searchsorted(np.cumsum([r * c // 64 for r, c in mods]), idx, side="right")
    assert np.all(np.diff(mod_of) >= 0)


def test_encode_deterministic():
    W, d = _small_module(seed=4, d_col=False)
    p = O.Params(C=64, P=8, b=4, S=8)
    a = _encode_module(W, d, p)[1]
    b = _encode_module(W, d, p)[1]
    for k in ("seed", "codes", "scale", "gain"):
        assert np.array_equal(a[k], b[k])


# ---------------------------------------------------------------- power-of-two scale
def test_pow2_scale_hand_values():
    # m = 3, qmax = 7: 7 * 2^-1 = 3.5 >= 3 > 7 * 2^-2 -> e = -1, q = rint(alpha / 0.5)
    q, f, sc = O.quantize(np.array([[3.0, -1.0, 0.2, 0.0]]), 4, O.SCALE_POW2)
    assert list(q[0]) == [6, -2, 0, 0] and int(f[0]) == 127 and sc[0] == 0.5
    # m exactly on qmax * 2^e keeps that e (no clipping needed): 3.5 = 7 * 2^-1
    q, f, sc = O.quantize(np.array([[3.5, 1.25]]), 4, O.SCALE_POW2)
    assert list(q[0]) == [7, 2] and int(f[0]) == 127
    # b = 3 (qmax 3): m = 10 -> 3 * 4 = 12 >= 10 > 6 -> e = 2
    q, f, sc = O.quantize(np.array([[10.0, -5.0]]), 3, O.SCALE_POW2)
    assert list(q[0]) == [2, -1] and int(f[0]) == 130 and sc[0] == 4.0
    # zero tile: all-zero record, field 0
    q, f, sc = O.quantize(np.zeros((1, 3)), 4, O.SCALE_POW2)
    assert not q.any() and int(f[0]) == 0 and sc[0] == 0.0


def test_pow2_scale_properties():
    rng = np.random.default_rng(3)
    for b in (2, 3, 4, 8):
        qmax = (1 << (b - 1)) - 1
        alpha = rng.standard_normal((400, 8)) * np.exp(rng.uniform(-20, 20, (400, 1)))
        q, f, sc = O.quantize(alpha, b, O.SCALE_POW2)
        m = np.abs(alpha).max(axis=1)
        e = f.astype(np.int64) - O.POW2_BIAS
        assert np.all(sc == np.ldexp(1.0, e))
        assert np.all(m <= qmax * sc) and np.all(m > qmax * sc / 2)   # smallest such e
        assert np.all(np.abs(alpha / sc[:, None]) <= qmax)             # nothing clips
        assert np.all(np.abs(q) <= qmax)
        assert np.all(np.abs(q).max(axis=1) >= (qmax + 1) // 2)
        assert np.array_equal(q, np.rint(alpha / sc[:, None]))


def test_pow2_paper_operating_point_record_and_stream():
    # AWSRC-P_F: (C, P, b, S) = (16, 4, 4, 16), ceil(log2 T) index, 8-bit exponent -> 7 bytes (Sec. 4)
    g = read_golden("paper_accounting.txt")
    N, K = int(g["n_scope"][0]), int(g["K"][0])
    p = O.Params(C=16, P=4, b=4, S=16, idx_bits=0, scale_fmt=O.SCALE_POW2)
    T = N // 16
    L = O.record_bytes(p, T)
    assert L == int(g["record_bytes"][0]) == 7
    assert O.header_bytes(108) + L * K == int(g["sidecar_bytes"][0])
    # a small stream in the same format: header fields and record size
    mods = [(4, 64)]
    rng = np.random.default_rng(1)
    T4 = 16
    enc = {"seed": rng.integers(0, 16, T4), "codes": rng.integers(-7, 8, (T4, 4)),
           "scale": rng.integers(0, 256, T4), "gain": rng.standard_normal(T4)}
    stream, K4, ne = O.build_stream(p, mods, enc, 64.0, per_module=False)
    hd = O.parse_header(stream)
    assert hd["scale_fmt"] == O.SCALE_POW2 and hd["scale_bits"] == 8 and hd["idx_bits"] == 4
    assert hd["L_rec"] == (4 + 4 + 16 + 8 + 7) // 8 == 4
    assert len(stream) == hd["h"] + K4 * 4 and K4 == ne == int(np.sum(enc["gain"] > 0))


def test_pow2_record_worked_example():
    g = read_golden("rec_v1_pow2_example.txt")
    codes = [int(c) for c in g["codes"]]
    rec = O.pack_record(int(g["idx"][0]), int(g["seed"][0]), codes, int(g["field"][0]), 28, 4, 4, 7,
                        scale_bits=O.SCALE_BITS_POW2)
    assert rec == bytes(int(x, 16) for x in g["bytes"])
    assert O.unpack_record(rec, 28, 4, 4, 4, O.SCALE_BITS_POW2) == (5, 9, codes, 125)


def test_pow2_decode_exact_power_of_two_scaling():
    # one record: r_hat = B_s (2^e q); orthonormal columns give |r_hat|^2 = 4^e |q|^2,
    # and every other tile of W0 is returned unchanged
    p = O.Params(C=16, P=4, b=4, S=16, idx_bits=0, scale_fmt=O.SCALE_POW2)
    mods = [(2, 32)]
    enc = {"seed": np.array([3, 0, 0, 0]), "codes": np.array([[7, -3, 0, 1]] + [[0] * 4] * 3),
           "scale": np.array([128 - 5, 0, 0, 0]), "gain": np.array([1.0, -1.0, -1.0, -1.0])}
    stream, K, _ = O.build_stream(p, mods, enc, 64.0, per_module=False)
    assert K == 1
    W0 = np.arange(64, dtype=np.float64).reshape(2, 32) / 7.0
    out = O.decode_add(stream, [W0])[0]
    rhat = out[0, :16] - W0[0, :16]
    assert math.isclose(float(rhat @ rhat), 4.0 ** -5 * (49 + 9 + 0 + 1), rel_tol=1e-12)
    assert np.array_equal(out[0, 16:], W0[0, 16:]) and np.array_equal(out[1], W0[1])


# ---------------------------------------------------------------- dense bf16 reconstruction
def test_rtn_dequant_reproduces_backbone_W0():
    rng = np.random.default_rng(8)
    W = (rng.standard_normal((6, 512)) * 0.02).astype(np.float32)
    W[0, :128] = 0.25                     # degenerate group
    for group in (64, 128, 256):
        codes, s16, z, W0 = O.rtn_backbone(W, group=group)
        assert np.array_equal(O.rtn_dequant(codes, s16, z, group), W0)


def test_bf16_round_matches_torch_on_fp32_values():
    import torch
    rng = np.random.default_rng(9)
    x = (rng.standard_normal(20000) * np.exp(rng.uniform(-30, 30, 20000))).astype(np.float32)
    # exact halfway points between bf16 neighbours, both parities
    base = np.array([1.0, 1.0078125, 3.0, -1.5], dtype=np.float32)
    x = np.concatenate([x, base + np.ldexp(1.0, -8).astype(np.float32) * np.abs(base)])
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(O.bf16_round(x.astype(np.float64)), want)


def test_reconstruct_bf16_empty_stream_is_rounded_backbone():
    rng = np.random.default_rng(10)
    W = (rng.standard_normal((4, 256)) * 0.02).astype(np.float32)
    codes, s16, z, W0 = O.rtn_backbone(W)
    p = O.Params(C=64, P=4, b=4, S=8)
    enc = {"seed": np.zeros(16, np.int64), "codes": np.zeros((16, 4), np.int64),
           "scale": np.zeros(16, np.int64), "gain": -np.ones(16)}
    stream, K, _ = O.build_stream(p, [(4, 256)], enc, 8.0, per_module=False)
    assert K == 0
    out = O.reconstruct_bf16(stream, [(codes, s16, z)])[0]
    assert np.array_equal(out, O.bf16_round(W0.astype(np.float64)))


# ------------------------------------------------------------------ SDQ (Sec. 3.3, Sec. 4)
def test_sdq_worked_example():
    """Hand-worked block in tests/golden/sdq_block_example.txt."""
    g = read_golden("sdq_block_example.txt")
    s16 = np.array([float(x) for x in g["scales"]], dtype=np.float16).view(np.uint16)
    codes, mean, step = O.sdq_encode(s16)
    assert codes.tolist() == [int(x) for x in g["codes"]]
    assert mean.tolist() == [float(g["mean"][0])]
    from fractions import Fraction
    assert step[0] == np.float32(float(Fraction(int(g["step_num"][0]), int(g["step_den"][0]))))


def _scale_sets(rng):
    yield rng.uniform(1e-3, 3e-3, 1000)                 # RTN g128 scales of N(0, 0.02^2) weights
    yield np.exp(rng.normal(-6.0, 1.0, 777))            # heavy spread, partial last block
    yield np.concatenate([np.full(256, 0.01), rng.uniform(1e-4, 1e-1, 300)])  # one constant block
    yield rng.choice([1e-3, 2e-3], 512)                 # two values


def test_sdq_error_bound_and_range():
    """Rounding to the nearest code: every dequantized scale lies within half a
    step of its scale (plus the float32 roundings of the mean, the deviation
    and the result), the codes stay in [-127, 127], and a block whose
    deviations are not all zero uses +-127 at its largest deviation."""
    rng = np.random.default_rng(11)
    for vals in _scale_sets(rng):
        s16 = vals.astype(np.float16).view(np.uint16)
        s = s16.view(np.float16).astype(np.float64)
        codes, mean, step = O.sdq_encode(s16)
        sh = O.sdq_scales(codes, mean, step).astype(np.float64)
        k = np.arange(s.size) // O.SDQ_BLOCK
        slack = 4 * np.finfo(np.float32).eps * np.maximum(np.abs(s), np.abs(mean[k].astype(np.float64)))
        assert np.all(np.abs(sh - s) <= 0.5 * step[k].astype(np.float64) + slack)
        assert codes.min() >= -127 and codes.max() <= 127
        for b in range(mean.size):
            cb = codes[b * O.SDQ_BLOCK:(b + 1) * O.SDQ_BLOCK]
            if step[b] > 0:
                assert np.abs(cb.astype(int)).max() == 127
            else:
                assert np.all(cb == 0)


def test_sdq_constant_block_is_exact_and_blocks_are_independent():
    rng = np.random.default_rng(12)
    base = np.concatenate([np.full(256, 0.0125), rng.uniform(1e-3, 3e-3, 256)]).astype(np.float16)
    codes, mean, step = O.sdq_encode(base.view(np.uint16))
    assert np.all(codes[:256] == 0) and step[0] == 0
    assert np.array_equal(O.sdq_scales(codes, mean, step)[:256], base[:256].astype(np.float32))
    other = base.copy()
    other[256:] = rng.uniform(1e-2, 2e-2, 256).astype(np.float16)
    c2, m2, s2 = O.sdq_encode(other.view(np.uint16))
    assert np.array_equal(c2[:256], codes[:256]) and m2[0] == mean[0] and s2[0] == step[0]


def test_rtn_dequant_sdq_reduces_to_rtn_when_scales_are_exact():
    """With every block constant, the SDQ scales equal the fp16 scales and the
    SDQ backbone is the RTN-v1 backbone bit for bit."""
    rng = np.random.default_rng(13)
    W = rng.normal(0, 0.02, (4, 256 * 128)).astype(np.float32)
    W[:, ::128] = 0.3      # same max in every group ...
    W[:, 1::128] = -0.3    # ... and min, so every scale is 0.04
    codes, s16, zero, W0 = O.rtn_backbone(W)
    sc, mu, st = O.sdq_encode(s16)
    assert np.all(sc == 0)
    assert np.array_equal(O.rtn_dequant_sdq(codes, zero, sc, mu, st), W0)


def test_reconstruct_bf16_sdq_reduces_to_fp16_path_when_scales_are_exact():
    """With every SDQ block constant the SDQ scales equal the fp16 ones, so the
    SDQ reconstruction of a stream with records equals the fp16-scale
    reconstruction (an independent path through rtn_dequant) bit for bit."""
    rng = np.random.default_rng(14)
    W = rng.normal(0, 0.02, (4, 128 * 128)).astype(np.float32)
    W[:, ::128] = 0.3
    W[:, 1::128] = -0.3
    codes, s16, zero, W0 = O.rtn_backbone(W)
    sc, mu, st = O.sdq_encode(s16)
    assert np.all(sc == 0)
    p = O.Params(C=64, P=4, b=4, S=8)
    T = 4 * 128 * 128 // 64
    enc = {"seed": rng.integers(0, 8, T), "codes": rng.integers(-7, 8, (T, 4)),
           "scale": np.full(T, 0x2000), "gain": rng.uniform(0, 1, T)}
    stream, K, _ = O.build_stream(p, [(4, 128 * 128)], enc, 0.05, per_module=False)
    assert K > 0
    a = O.reconstruct_bf16_sdq(stream, [(codes, zero, sc, mu, st)])[0]
    b = O.reconstruct_bf16(stream, [(codes, s16, zero)])[0]
    assert np.array_equal(a, b)


def test_reconstruct_bf16_sdq_changes_only_record_tiles():
    """Against the rounded SDQ backbone, a stream changes exactly the tiles it
    holds records for (each by its correction B_s scale q, checked through the
    norm identity of the orthonormal columns before rounding)."""
    rng = np.random.default_rng(15)
    W = rng.normal(0, 0.02, (3, 512)).astype(np.float32)
    codes, s16, zero, _ = O.rtn_backbone(W)
    sc, mu, st = O.sdq_encode(s16)
    W0s = O.rtn_dequant_sdq(codes, zero, sc, mu, st).astype(np.float64)
    p = O.Params(C=64, P=4, b=4, S=8)
    T = 3 * 512 // 64
    gain = -np.ones(T)
    gain[[2, 17]] = [2.0, 1.0]
    enc = {"seed": np.full(T, 5), "codes": np.tile([3, -2, 0, 7], (T, 1)),
           "scale": np.full(T, 0x3C00), "gain": gain}   # fp16 1.0
    stream, K, _ = O.build_stream(p, [(3, 512)], enc, 64.0, per_module=False)
    assert K == 2
    out = O.reconstruct_bf16_sdq(stream, [(codes, zero, sc, mu, st)])[0]
    base = O.bf16_round(W0s)
    changed = {int(t) for t in np.nonzero((out != base).reshape(T, 64).any(axis=1))[0]}
    assert changed <= {2, 17} and changed
    exact = O.decode_add(stream, [W0s])[0] - W0s
    for t in (2, 17):
        r = exact.reshape(T, 64)[t]
        assert math.isclose(float(r @ r), 9 + 4 + 0 + 49, rel_tol=1e-12)  # scale 1, orthonormal B_s


def test_sdq_rate():
    """8 bits per group and 64 per block of 256: 0.0645 bits per weight at
    g128, against 0.125 for the fp16 scales (Sec. 4 reports 0.068 for its
    format, which it does not specify)."""
    n_w = 2048 * 11008
    n_g = n_w // 128
    assert abs(O.sdq_bits_per_weight(n_w, n_g) - (8 + 64 / 256) / 128) < 1e-12
    assert abs(16 * n_g / n_w - 0.125) < 1e-12


# ------------------------------------------------ parity exemptions (flags)
# The GPU parity tests skip the bit-exact code/scale comparison only where
# the oracle flags a knife edge; these pins fix what the flags may cover.
def test_boundary_flags_hand_values():
    """A coefficient flags its tile exactly when |alpha*/scale| lies within
    1e-9 of a rounding midpoint n + 1/2 below qmax + 1/2 (Sec. 3.2 RTN)."""
    qmax = 7
    sc = np.array([1.0])
    cases = [
        (2.5, True),                  # on the midpoint
        (-2.5, True),                 # sign does not matter
        (2.5 + 5e-10, True),          # just inside, above
        (2.5 - 5e-10, True),          # just inside, below
        (2.5 + 3e-9, False),          # just outside
        (2.5 - 3e-9, False),
        (2.25, False), (3.0, False), (0.0, False),
        (7.5, False),                 # beyond qmax + 1/2: clamps either way
        (9.5, False),
        (6.5, True),                  # the last midpoint below qmax + 1/2
    ]
    for a, want in cases:
        alpha = np.array([[0.25, a, 0.0, 1.0]])
        assert bool(O._boundary_flags(alpha, sc, qmax)[0]) == want, a
    # the scale divides: alpha = 0.625 with scale 0.25 is the midpoint 2.5
    assert O._boundary_flags(np.array([[0.625]]), np.array([0.25]), qmax)[0]
    assert not O._boundary_flags(np.array([[0.6]]), np.array([0.25]), qmax)[0]
    # a zero scale (empty record) is never flagged
    assert not O._boundary_flags(np.array([[0.5]]), np.array([0.0]), qmax)[0]


def test_boundary_flags_cover_every_code_flip():
    """Perturbing alpha* by 5e-10 of the scale (far above the fp64 re-score's
    error, below the flag's tolerance) changes a code only on flagged tiles;
    unflagged tiles keep their codes."""
    rng = np.random.default_rng(123)
    qmax, n = 7, 4000
    sc = np.exp(rng.normal(-6, 1, n))
    x = rng.uniform(-7.4, 7.4, (n, 8))
    x[: n // 4, 3] = rng.integers(-7, 7, n // 4) + 0.5 + rng.uniform(-4e-10, 4e-10, n // 4)  # near midpoints
    alpha = x * sc[:, None]
    flags = O._boundary_flags(alpha, sc, qmax)
    q0 = np.clip(np.rint(alpha / sc[:, None]), -qmax, qmax)
    changed = np.zeros(n, bool)
    for sgn in (-1.0, 1.0):
        q1 = np.clip(np.rint((alpha + sgn * 5e-10 * sc[:, None]) / sc[:, None]), -qmax, qmax)
        changed |= np.any(q1 != q0, axis=1)
    assert flags[: n // 4].all()
    assert not np.any(changed & ~flags)
    assert not flags[n // 4:].any()


def test_scale_flags_fp16_hand_values():
    """fp16 scales: flagged exactly when m/qmax lies within 1e-12 (relative)
    of an fp32 rounding midpoint, where the first of the two roundings of
    f16(f32(m/qmax)) could go either way."""
    qmax = 7
    mid = 1.0 + 2.0 ** -24            # halfway between 1 and the next fp32
    for v, want in [(mid, True), (mid + 2.0 ** -42, True), (mid - 2.0 ** -42, True),
                    (mid + 2.0 ** -36, False), (mid - 2.0 ** -36, False),
                    (1.0, False), (1.1, False), (0.75 + 2.0 ** -25, True), (0.75 + 3 * 2.0 ** -25, True), (0.75 + 2.0 ** -26, False)]:
        alpha = np.array([[v * qmax, -0.5]])
        assert bool(O._scale_flags(alpha, qmax)[0]) == want, v
    assert not O._scale_flags(np.zeros((1, 4)), qmax)[0]


def test_scale_flags_fp16_cover_every_rounding_flip():
    """A relative perturbation of 1e-13 of m changes f32(m/qmax) only on
    flagged tiles."""
    rng = np.random.default_rng(7)
    qmax, n = 7, 20000
    v = np.exp(rng.normal(-7, 2, n))
    f = v.astype(np.float32).astype(np.float64)
    ulp = np.spacing(f.astype(np.float32)).astype(np.float64)
    v[: n // 10] = (f + 0.5 * ulp)[: n // 10] * (1 + rng.uniform(-1e-14, 1e-14, n // 10))
    alpha = np.stack([v * qmax, -0.5 * v * qmax], axis=1)
    flags = O._scale_flags(alpha, qmax)
    base = (alpha[:, 0] / qmax).astype(np.float32)
    changed = np.zeros(n, bool)
    for r in (1 - 1e-13, 1 + 1e-13):
        changed |= ((alpha[:, 0] * r) / qmax).astype(np.float32) != base
    assert flags[: n // 10].all()
    assert changed[: n // 10].any()
    assert not np.any(changed & ~flags)
    assert flags[n // 10:].mean() < 1e-3


def test_scale_flags_pow2_hand_values():
    """Power-of-two scales: flagged exactly when m/qmax lies within 1e-12
    (relative) of a power of two, where the exponent rule of Sec. 3.2 could
    go either way."""
    qmax = 7
    for v, want in [(2.0 ** -5, True), (2.0 ** -5 * (1 + 1e-13), True), (2.0 ** -5 * (1 - 1e-13), True),
                    (2.0 ** -5 * (1 + 1e-11), False), (2.0 ** -5 * (1 - 1e-11), False),
                    (3.0 * 2.0 ** -6, False), (1.0, True)]:
        alpha = np.array([[0.0, -v * qmax]])
        assert bool(O._scale_flags(alpha, qmax, scale_fmt=O.SCALE_POW2)[0]) == want, v
    assert not O._scale_flags(np.zeros((1, 2)), qmax, scale_fmt=O.SCALE_POW2)[0]


@pytest.mark.parametrize("fmt,gen", [(O.SCALE_FP16, 1), (O.SCALE_POW2, 1), (O.SCALE_FP16, 2)])
def test_candidate_matches_the_batched_search(fmt, gen):
    """candidate() (one tile, one seed; used to check the GPU's record when it
    picks a tied seed) equals the batched search's column for that seed, and
    its codes and scale at the chosen seed are the search's record."""
    rng = np.random.default_rng(31 + fmt + 10 * gen)
    op = O.Params(C=32, P=5, b=4, S=12, basis_key=99, ridge_lambda=1e-6, scale_fmt=fmt, gen_version=gen)
    R = rng.normal(0, 0.01, (6, 32))
    D = np.exp(rng.normal(0, 1.5, (6, 32)))
    out = O.encode_tiles(R, D, op, keep_all=True)
    for i in range(6):
        for s in range(op.S):
            q, bits, g, alpha = O.candidate(R[i], D[i], op, s)
            # same fp64 steps, batched or not: agreement to rounding order
            assert abs(g - out["all_gains"][i, s]) <= 1e-12 * out["energy"][i]
            if s == out["seed"][i]:
                assert np.array_equal(q, out["codes"][i]) and bits == out["scale"][i]
                assert np.allclose(alpha, out["alpha"][i], rtol=1e-12, atol=0)
