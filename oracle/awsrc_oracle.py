"""AWSRC reference oracle.  TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct CPU implementation of what the AWSRC
encoder/decoder hot path computes, in numpy float64 (the backbone quantizer is
emulated bit-exactly in numpy float32, the precision its recipe fixes).  Only
the test-suite, the package smoke check and the benchmark's CPU-baseline leg
may import this module; the product path (the HIP library and its Python
binding) never does, and this module imports nothing from the product.

Paper map (arXiv 2608.23144, "Activation-Weighted Seeded Residual Coding"):

* Eq. (1), Sec. 3.1  backbone, residual and repaired weight: W0 = Q(W),
  R = W - W0, W_hat = W0 + R_hat; R is cut into row-wise tiles r_t of length C.
* Eq. (2), Sec. 3.1  B_s = GenBasis(s, C, P): normalized Hadamard columns with
  a seeded sign pattern and a seeded choice of P columns.
* Eq. (3), Sec. 3.2  activation-weighted ridge least squares for alpha*_{t,s}.
* Sec. 3.2            coefficient-wise b-bit RTN with one scale per tile; each
  tile keeps the seed whose rounded coefficients leave the least weighted error.
* Eq. (4), Sec. 3.3  byte-normalized gain rho_t; non-positive records are
  dropped; per-module quotas (U variant) or one global ranking (P variant)
  whose record-boundary prefixes all decode.
* Eq. (5), Sec. 3.4  serialized rate: header plus fixed-size records.

Readings of points the paper leaves open (each listed in the design notes):

* GEN-v1 generator: splitmix64 counter stream keyed by ``basis_key``; word i
  of seed s is output number s*2^32 + i; sign bit j is bit (j mod 64) of word
  floor(j/64); column p uses word ceil(C/64)+p mapped to [0, C-p) by Lemire's
  multiply-shift on its high 32 bits and takes the m-th smallest unused
  column.  The seeded coordinate permutation of Sec. 3.1 is not applied
  (generator version 1).
* Hadamard matrix: Sylvester natural order, H[j, c] = (-1)^popcount(j & c),
  scaled by 1/sqrt(C).
* Ridge constant: eps_t = lambda * mean_j d_{t,j}; it enters the fit only,
  not the selection score.
* SDQ of the backbone's group scales (Sec. 3.3, Sec. 4 give only its name,
  origin and size): blocks of 256 group scales, an int8 code per scale
  around the block mean with one float32 mean and step per block
  (``sdq_encode``).
* Scale, two formats (Sec. 3.2 names one power-of-two scale per tile stored
  as an exponent of width b_e, Eq. (5); the default here is fp16):
  - fp16: scale16 = f16(f32(m / qmax)) with both roundings to nearest even,
    m = max_p |alpha*_p|; a zero m, or a scale that rounds to zero, gives an
    all-zero record with gain 0; fp16 overflow saturates at 65504;
  - pow2: scale = 2^e with e the smallest integer such that m <= qmax 2^e
    (no code clips), clamped to [-128, 127] and stored as e + 128 in
    b_e = 8 bits; m = 0 gives an all-zero record (field 0, gain 0).
  Codes q_p = clip(rint(alpha*_p / scale), +-qmax), qmax = 2^(b-1) - 1.
* Ties: the lowest seed wins among exactly equal gains; equal rho orders by
  the lower global tile index; only gain > 0 is eligible.
* Backbone RTN-v1: asymmetric INT4, groups of 128 input columns, fp32
  arithmetic with correctly rounded division (see ``rtn_backbone``).
* REC-v1 / STREAM-v1 byte layouts: see ``pack_record`` and ``stream_header``.
"""
from __future__ import annotations

import functools
import math
import struct
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

MASK64 = (1 << 64) - 1
GOLDEN_GAMMA = 0x9E3779B97F4A7C15
MAGIC = b"AWSR"
STREAM_VERSION = 1
HEADER_FIXED_BYTES = 40
SCALE_FP16, SCALE_POW2 = 0, 1
SCALE_BITS_FP16 = 16
SCALE_BITS_POW2 = 8          # b_e of Eq. (5) for the power-of-two scale
POW2_BIAS = 128
FP16_MAX = 65504.0


# --------------------------------------------------------------------------
# Parameters
# --------------------------------------------------------------------------
@dataclass(frozen=True)
class Params:
    """(C, P, b, S) of Sec. 3.1 plus the generator key, ridge factor and index width."""
    C: int
    P: int
    b: int
    S: int
    basis_key: int = 0
    ridge_lambda: float = 1e-6
    idx_bits: int = 32          # 0 selects ceil(log2 T_total) as in Eq. (5)
    gen_version: int = 1
    scale_fmt: int = SCALE_FP16  # SCALE_FP16 or SCALE_POW2

    @property
    def scale_bits(self) -> int:
        return SCALE_BITS_POW2 if self.scale_fmt == SCALE_POW2 else SCALE_BITS_FP16

    @property
    def qmax(self) -> int:
        return (1 << (self.b - 1)) - 1


# --------------------------------------------------------------------------
# Seeded basis, Eq. (2)
# --------------------------------------------------------------------------
def splitmix64(key: int, n: int) -> int:
    """Output number n (n >= 0) of the splitmix64 generator started at state `key`.

    The state advances by the golden-ratio increment before each output and
    the output is the state passed through the variant-13 mixing function
    (Steele, Lea & Flood, OOPSLA 2014; Vigna's public-domain reference).
    """
    z = (key + (n + 1) * GOLDEN_GAMMA) & MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def basis_word(key: int, s: int, i: int) -> int:
    """Word i of seed s: one counter stream per seed, 2^32 words apart."""
    return splitmix64(key, (s << 32) + i)


def gen_basis(key: int, s: int, C: int, P: int) -> Tuple[np.ndarray, List[int]]:
    """GenBasis(s, C, P) of Eq. (2), generator version 1.

    Returns the sign pattern sigma in {+1, -1}^C and the P distinct selected
    Hadamard columns in draw order.
    """
    n_sign_words = (C + 63) // 64
    sigma = np.empty(C, dtype=np.int64)
    for j in range(C):
        w = basis_word(key, s, j // 64)
        sigma[j] = 1 - 2 * ((w >> (j % 64)) & 1)
    unused = list(range(C))
    cols: List[int] = []
    for p in range(P):
        v = basis_word(key, s, n_sign_words + p)
        m = ((v >> 32) * (C - p)) >> 32          # Lemire multiply-shift into [0, C-p)
        cols.append(unused.pop(m))               # m-th smallest column not yet drawn
    return sigma, cols


def gen_permutation(key: int, s: int, C: int, P: int) -> np.ndarray:
    """Seeded coordinate permutation of generator version 2 (the permutation of
    Eq. (2)'s basis, Sec. 3.1): coordinate j draws the sort key word
    ceil(C/64) + P + j of seed s (after the sign and column words), and
    pi(j) is the rank of (key_j, j) in increasing order.  Ranking independent
    uniform keys gives a uniform permutation (the random-keys shuffle)."""
    n_sign_words = (C + 63) // 64
    keys = [basis_word(key, s, n_sign_words + P + j) for j in range(C)]
    order = sorted(range(C), key=lambda j: (keys[j], j))
    pi = np.empty(C, dtype=np.int64)
    for r, j in enumerate(order):
        pi[j] = r
    return pi


def hadamard(C: int) -> np.ndarray:
    """Order-C Sylvester Hadamard matrix in natural order (integer entries +-1)."""
    return _hadamard(C).copy()


@functools.lru_cache(maxsize=None)
def _hadamard(C: int) -> np.ndarray:
    assert C >= 1 and C & (C - 1) == 0, "C must be a power of two"
    H = np.empty((C, C), dtype=np.int64)
    for j in range(C):
        for c in range(C):
            H[j, c] = -1 if bin(j & c).count("1") % 2 else 1
    H.setflags(write=False)
    return H


def basis_matrix(key: int, s: int, C: int, P: int, gen_version: int = 1) -> np.ndarray:
    """B_s in R^{C x P} (Eq. (2)): B[j, p] = sigma_j H[pi(j), c_p] / sqrt(C),
    with pi the identity for generator version 1 and the seeded coordinate
    permutation for version 2 (signs and columns are the same words in both)."""
    if gen_version not in (1, 2):
        raise ValueError("unsupported generator version")
    sigma, cols = gen_basis(key, s, C, P)
    H = _hadamard(C)
    rows = gen_permutation(key, s, C, P) if gen_version == 2 else np.arange(C)
    return (sigma[:, None] * H[rows][:, cols]).astype(np.float64) / math.sqrt(C)


# --------------------------------------------------------------------------
# Backbone Q of Eq. (1): RTN-v1, asymmetric INT4 with groups of 128 inputs
# --------------------------------------------------------------------------
def rtn_backbone(W32: np.ndarray, group: int = 128):
    """RTN-INT4 backbone W0 = Q(W) (Eq. (1); Sec. 4 uses RTN with group size 128).

    All arithmetic is IEEE float32 with round-to-nearest-even and correctly
    rounded division, per group of `group` consecutive input columns:
        s32 = (max - min) / 15;  s16 = f16(s32) (saturating);  s = f32(s16)
        z = clip(rint(-min / s), 0, 15);  q = clip(rint(w / s) + z, 0, 15)
        W0 = f32(q - z) * s
    A group whose s16 is zero is stored as s16 = 1.0, z = 0, q = 0 (W0 = 0).

    Returns (codes u8 [rows, cols/2] with the even column in the low nibble,
    scale u16 fp16 bits [rows, cols/group], zero u8 [rows, cols/group],
    W0 float32 [rows, cols]).
    """
    W32 = np.ascontiguousarray(W32, dtype=np.float32)
    rows, cols = W32.shape
    assert cols % group == 0 and group % 2 == 0
    Wg = W32.reshape(rows, cols // group, group)
    mn = Wg.min(axis=2)
    mx = Wg.max(axis=2)
    s32 = (mx - mn) / np.float32(15.0)
    with np.errstate(over="ignore"):
        s16 = s32.astype(np.float16)
    s16 = np.where(np.isinf(s16), np.float16(FP16_MAX), s16)
    degenerate = s16 == 0
    s16 = np.where(degenerate, np.float16(1.0), s16)
    s = s16.astype(np.float32)
    z = np.clip(np.rint(-mn / s), np.float32(0), np.float32(15))
    q = np.clip(np.rint(Wg / s[..., None]) + z[..., None], np.float32(0), np.float32(15))
    z = np.where(degenerate, np.float32(0), z)
    q = np.where(degenerate[..., None], np.float32(0), q)
    W0 = (q - z[..., None]).astype(np.float32) * s[..., None]
    qi = q.astype(np.uint8).reshape(rows, cols)
    codes = (qi[:, 0::2] | (qi[:, 1::2] << 4)).astype(np.uint8)
    return (codes, s16.view(np.uint16).copy(), z.astype(np.uint8),
            W0.reshape(rows, cols).astype(np.float32))


def rtn_dequant(codes: np.ndarray, scale16: np.ndarray, zero: np.ndarray, group: int = 128) -> np.ndarray:
    """W0 from the stored backbone (codes, fp16 scale bits, zero points):
    W0 = f32(q - z) * s per group, the last step of RTN-v1, in float32."""
    codes = np.asarray(codes, dtype=np.uint8)
    rows = codes.shape[0]
    cols = codes.shape[1] * 2
    q = np.empty((rows, cols), dtype=np.float32)
    q[:, 0::2] = codes & 0x0F
    q[:, 1::2] = codes >> 4
    s = np.asarray(scale16, dtype=np.uint16).view(np.float16).astype(np.float32)
    z = np.asarray(zero, dtype=np.float32)
    qg = q.reshape(rows, cols // group, group)
    return ((qg - z[..., None]) * s[..., None]).astype(np.float32).reshape(rows, cols)


SDQ_BLOCK = 256


def sdq_encode(scale16: np.ndarray, block: int = SDQ_BLOCK):
    """Scale double quantization (SDQ) of the RTN group scales (Sec. 3.3 names
    it, after QLoRA's double quantization of the quantization constants, and
    Sec. 4 gives its size for RTN g128: 0.068 instead of 0.125 bits per weight).
    Reading: the fp16 group scales, flattened in row-major order, are cut into
    blocks of `block` consecutive groups (the last block may be shorter); per
    block of n scales s_g
        mu    = f32(sum_g s_g / n)    (the sum in float64, g in order; one division)
        dlt_g = f32(s_g - mu)         (one float32 rounding)
        a     = max_g |dlt_g|
        c_g   = rint(dlt_g * 127 / a) in [-127, 127] (float64: the product is
                exact, one division, ties to even); every c_g = 0 when a = 0
        step  = f32(a / 127)          (float64 division, one rounding)
    stored as one int8 code per group and two float32 (mu, step) per block:
    8 + 64 / block bits per group (0.0645 bits per weight at g128, block 256).
    Returns (codes int8 [n_groups], mean float32 [n_blocks], step float32 [n_blocks])."""
    s = np.asarray(scale16, dtype=np.uint16).reshape(-1).view(np.float16).astype(np.float64)
    n = s.size
    nblk = (n + block - 1) // block
    codes = np.zeros(n, dtype=np.int8)
    mean = np.zeros(nblk, dtype=np.float32)
    step = np.zeros(nblk, dtype=np.float32)
    for k in range(nblk):
        sb = s[k * block:(k + 1) * block]
        tot = 0.0
        for v in sb:  # float64, in order
            tot += float(v)
        mu = np.float32(tot / len(sb))
        dlt = (sb.astype(np.float32) - mu).astype(np.float32)
        a = float(np.abs(dlt).max())
        if a > 0.0:
            c = np.rint(dlt.astype(np.float64) * 127.0 / a)
            codes[k * block:k * block + len(sb)] = np.clip(c, -127, 127).astype(np.int8)
        mean[k] = mu
        step[k] = np.float32(a / 127.0)
    return codes, mean, step


def sdq_scales(codes: np.ndarray, mean: np.ndarray, step: np.ndarray, block: int = SDQ_BLOCK) -> np.ndarray:
    """Dequantized group scales s_hat_g = f32(mu + c_g * step) of the group's
    block (float64 sum of exact terms, one rounding to float32)."""
    c = np.asarray(codes, dtype=np.int8).reshape(-1).astype(np.float64)
    k = np.arange(c.size) // block
    return (np.asarray(mean, np.float32)[k].astype(np.float64)
            + c * np.asarray(step, np.float32)[k].astype(np.float64)).astype(np.float32)


def rtn_dequant_sdq(codes: np.ndarray, zero: np.ndarray, sdq_codes: np.ndarray, sdq_mean: np.ndarray,
                    sdq_step: np.ndarray, group: int = 128) -> np.ndarray:
    """W0 of an RTN-INT4-SDQ backbone: W0 = f32(q - z) * s_hat per group, the
    RTN-v1 codes and zero points with the SDQ-dequantized scales."""
    codes = np.asarray(codes, dtype=np.uint8)
    rows = codes.shape[0]
    cols = codes.shape[1] * 2
    q = np.empty((rows, cols), dtype=np.float32)
    q[:, 0::2] = codes & 0x0F
    q[:, 1::2] = codes >> 4
    sh = sdq_scales(sdq_codes, sdq_mean, sdq_step).reshape(rows, cols // group)
    z = np.asarray(zero, dtype=np.float32)
    qg = q.reshape(rows, cols // group, group)
    return ((qg - z[..., None]) * sh[..., None]).astype(np.float32).reshape(rows, cols)


def sdq_bits_per_weight(n_weights: int, n_groups: int, block: int = SDQ_BLOCK) -> float:
    """Scale metadata rate of SDQ: 8 bits per group plus 64 per block."""
    return (8 * n_groups + 64 * ((n_groups + block - 1) // block)) / n_weights


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 (8 significant bits, ties
    to even), returned as float64; one rounding of the exact value."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                    # x = m 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.rint(m * 256.0) / 256.0, e)


def reconstruct_bf16(stream: bytes, backbones: Sequence[Tuple[np.ndarray, np.ndarray, np.ndarray]],
                     group: int = 128) -> List[np.ndarray]:
    """Dense bf16 repaired weights (the evaluation form of Sec. 4): each
    module's W0 dequantized from its stored backbone, the stream's
    corrections added (decode_add), and the exact sum rounded to bfloat16."""
    W0s = [rtn_dequant(c, s, z, group) for c, s, z in backbones]
    return [bf16_round(w) for w in decode_add(stream, W0s)]


def reconstruct_bf16_sdq(stream: bytes, backbones: Sequence[Tuple[np.ndarray, np.ndarray, np.ndarray, np.ndarray,
                                                                     np.ndarray]],
                         group: int = 128) -> List[np.ndarray]:
    """Dense bf16 repaired weights on the RTN-INT4-SDQ backbone (the backbone
    Sec. 4 evaluates with the codecs): each module's W0 dequantized from its
    codes, zero points and SDQ scale codes (codes, zero, sdq_codes, sdq_mean,
    sdq_step per module, as rtn_dequant_sdq takes them), the stream's
    corrections added (decode_add), and the exact sum rounded to bfloat16."""
    W0s = [rtn_dequant_sdq(c, z, sc, mu, st, group) for c, z, sc, mu, st in backbones]
    return [bf16_round(w) for w in decode_add(stream, W0s)]


def residual(W32: np.ndarray, W0: np.ndarray) -> np.ndarray:
    """R = W - W0 of Eq. (1), one float32 subtraction per element."""
    return (np.asarray(W32, dtype=np.float32) - np.asarray(W0, dtype=np.float32)).astype(np.float32)


# --------------------------------------------------------------------------
# Tiles (Sec. 3.1): row-wise runs of C consecutive input coordinates
# --------------------------------------------------------------------------
def tiles(A: np.ndarray, C: int) -> np.ndarray:
    """[rows, cols] -> [rows*cols/C, C]; tile t = row*(cols/C) + block."""
    rows, cols = A.shape
    assert cols % C == 0
    return np.ascontiguousarray(A).reshape(rows * (cols // C), C)


def tile_weights(d: np.ndarray, rows: int, cols: int, C: int) -> np.ndarray:
    """Coordinate weights d_{t,j} per tile: a [cols] activation vector is shared by
    every row (Sec. 3.2); a [rows, cols] blended diagonal is row specific."""
    d = np.asarray(d, dtype=np.float64)
    if d.ndim == 1:
        assert d.shape[0] == cols
        return np.tile(d.reshape(cols // C, C), (rows, 1))
    assert d.shape == (rows, cols)
    return d.reshape(rows * (cols // C), C)


# --------------------------------------------------------------------------
# Fit, quantize, score (Eq. (3), Sec. 3.2, Eq. (4))
# --------------------------------------------------------------------------
def fit(R: np.ndarray, Dw: np.ndarray, B: np.ndarray, ridge_lambda: float):
    """alpha*_{t,s} = argmin_a sum_j d_j ([B a]_j - r_j)^2 + eps_t |a|^2   (Eq. (3)).

    Normal equations (B^T D B + eps I) a = B^T D r, solved per tile with
    LAPACK's LU solver; eps_t = lambda * mean_j d_{t,j}.
    Returns (alpha*, G = B^T D B + eps I, b = B^T D r).
    """
    N, C = R.shape
    P = B.shape[1]
    BB = (B[:, :, None] * B[:, None, :]).reshape(C, P * P)
    G = (Dw @ BB).reshape(N, P, P)
    eps = ridge_lambda * Dw.mean(axis=1)
    G = G + eps[:, None, None] * np.eye(P)[None]
    bvec = (Dw * R) @ B
    alpha = np.linalg.solve(G, bvec[..., None])[..., 0]
    return alpha, G, bvec


def pow2_exponent(m: float, qmax: int) -> int:
    """Smallest integer e with m <= qmax * 2^e (m > 0), by exact comparisons."""
    e = math.frexp(m / qmax)[1]          # m/qmax < 2^e, up to the rounding of the division
    while m > qmax * math.ldexp(1.0, e):
        e += 1
    while m <= qmax * math.ldexp(1.0, e - 1):
        e -= 1
    return e


def quantize(alpha: np.ndarray, b: int, scale_fmt: int = SCALE_FP16):
    """Coefficient-wise b-bit RTN with one scale per tile (Sec. 3.2).

    Returns (codes int64 [N, P], stored scale field uint16 [N] (fp16 bits, or
    the biased exponent), scale value float64 [N]).
    """
    qmax = (1 << (b - 1)) - 1
    m = np.abs(alpha).max(axis=1)
    if scale_fmt == SCALE_POW2:
        e = np.array([min(127, max(-128, pow2_exponent(float(v), qmax))) if v > 0 else -POW2_BIAS for v in m],
                     dtype=np.int64)
        sc = np.ldexp(1.0, e)
        empty = m == 0
        q = np.clip(np.rint(alpha / sc[:, None]), -qmax, qmax)
        q = np.where(empty[:, None], 0.0, q).astype(np.int64)
        bits = (e + POW2_BIAS).astype(np.uint16)
        sc = np.where(empty, 0.0, sc)
        return q, bits, sc
    s32 = (m / qmax).astype(np.float32)
    with np.errstate(over="ignore"):
        s16 = s32.astype(np.float16)
    s16 = np.where(np.isinf(s16), np.float16(FP16_MAX), s16)
    sc = s16.astype(np.float64)
    empty = (m == 0) | (sc == 0)
    safe = np.where(empty, 1.0, sc)
    q = np.clip(np.rint(alpha / safe[:, None]), -qmax, qmax)
    q = np.where(empty[:, None], 0.0, q).astype(np.int64)
    bits = np.where(empty, np.uint16(0), s16.view(np.uint16)).astype(np.uint16)
    sc = np.where(empty, 0.0, sc)
    return q, bits, sc


def weighted_gain(R: np.ndarray, Dw: np.ndarray, Rhat: np.ndarray) -> np.ndarray:
    """Numerator of Eq. (4): sum_j d_j [r_j^2 - (r_j - rhat_j)^2]."""
    return np.sum(Dw * (R * R - (R - Rhat) ** 2), axis=1)


def _boundary_flags(alpha, sc, qmax, tol=1e-9):
    """True where some alpha*_p / scale lies within tol of a rounding midpoint."""
    safe = np.where(sc == 0, 1.0, sc)
    x = np.abs(alpha / safe[:, None])
    frac = np.abs(x - np.floor(x) - 0.5)
    return np.any((frac < tol) & (x < qmax + 0.5), axis=1) & (sc > 0)


def _scale_flags(alpha, qmax, tol=1e-12, scale_fmt=SCALE_FP16):
    """True where the scale choice is on a knife edge: m/qmax within tol
    (relative) of an fp32 rounding midpoint (fp16 format), or of a power of
    two (pow2 format)."""
    m = np.abs(alpha).max(axis=1)
    if scale_fmt == SCALE_POW2:
        v = m / qmax
        lg = np.log2(np.where(m > 0, v, 1.0))
        return (np.abs(lg - np.rint(lg)) <= tol / math.log(2)) & (m > 0)
    v = m / qmax
    f = v.astype(np.float32).astype(np.float64)
    ulp = np.spacing(np.abs(v).astype(np.float32)).astype(np.float64)
    mid_dist = np.abs(np.abs(v - f) - 0.5 * ulp)
    return (mid_dist <= tol * np.maximum(np.abs(v), 1e-300)) & (m > 0)


def encode_tiles(R: np.ndarray, Dw: np.ndarray, params: Params,
                 bases: Optional[Sequence[np.ndarray]] = None,
                 quantize_coeffs: bool = True, keep_all: bool = False) -> Dict[str, np.ndarray]:
    """Seeded fit + quantize + select for every tile (Sec. 3.2).

    R, Dw: [N, C] residual tiles and their coordinate weights.  For every seed
    s in 0..S-1 (or every explicit basis in `bases`) the tile is fitted
    (Eq. (3)), the coefficients are quantized, and the weighted gain of the
    quantized reconstruction (Eq. (4) numerator) is evaluated; the seed with
    the largest gain (= least weighted error after rounding) is kept, the
    lowest seed winning exact ties.  With quantize_coeffs=False the
    unquantized fit is scored instead (used by the exact-reconstruction check).
    """
    R = np.asarray(R, dtype=np.float64)
    Dw = np.asarray(Dw, dtype=np.float64)
    N, C = R.shape
    P = params.P
    qmax = params.qmax
    if bases is None:
        bases = [basis_matrix(params.basis_key, s, C, P, params.gen_version) for s in range(params.S)]
    n_seeds = len(bases)
    best_gain = np.full(N, -np.inf)
    second_gain = np.full(N, -np.inf)
    best_seed = np.zeros(N, dtype=np.int64)
    best_codes = np.zeros((N, P), dtype=np.int64)
    best_bits = np.zeros(N, dtype=np.uint16)
    best_sc = np.zeros(N)
    best_alpha = np.zeros((N, P))
    all_gains = np.empty((N, n_seeds)) if keep_all else None
    for s, B in enumerate(bases):
        alpha, _, _ = fit(R, Dw, B, params.ridge_lambda)
        if quantize_coeffs:
            q, bits, sc = quantize(alpha, params.b, params.scale_fmt)
            ahat = sc[:, None] * q
        else:
            q = np.zeros((N, P), dtype=np.int64)
            bits = np.zeros(N, dtype=np.uint16)
            sc = np.zeros(N)
            ahat = alpha
        g = weighted_gain(R, Dw, ahat @ B.T)
        if keep_all:
            all_gains[:, s] = g
        better = g > best_gain
        second_gain = np.where(better, best_gain, np.maximum(second_gain, g))
        best_gain = np.where(better, g, best_gain)
        best_seed = np.where(better, s, best_seed)
        best_codes = np.where(better[:, None], q, best_codes)
        best_bits = np.where(better, bits, best_bits)
        best_sc = np.where(better, sc, best_sc)
        best_alpha = np.where(better[:, None], alpha, best_alpha)
    energy = np.sum(Dw * R * R, axis=1)
    out = {
        "seed": best_seed, "codes": best_codes, "scale": best_bits, "scale_value": best_sc,
        "gain": best_gain, "alpha": best_alpha, "energy": energy,
        "flag_half": _boundary_flags(best_alpha, best_sc, qmax) if quantize_coeffs else np.zeros(N, bool),
        "flag_scale": (_scale_flags(best_alpha, qmax, scale_fmt=params.scale_fmt) if quantize_coeffs
                       else np.zeros(N, bool)),
        "flag_tie": (best_gain - second_gain) <= 1e-6 * np.abs(best_gain),
        "flag_zero": np.abs(best_gain) <= 1e-12 * energy,
    }
    if keep_all:
        out["all_gains"] = all_gains
    return out


def candidate(R_t: np.ndarray, D_t: np.ndarray, params: Params, s: int):
    """The full encoder chain for one (tile, seed): (codes, scale bits, gain, alpha*)."""
    B = basis_matrix(params.basis_key, s, R_t.shape[0], params.P, params.gen_version)
    alpha, _, _ = fit(R_t[None].astype(np.float64), D_t[None].astype(np.float64), B, params.ridge_lambda)
    q, bits, sc = quantize(alpha, params.b, params.scale_fmt)
    g = weighted_gain(R_t[None].astype(np.float64), D_t[None].astype(np.float64), (sc[:, None] * q) @ B.T)
    return q[0], int(bits[0]), float(g[0]), alpha[0]


# --------------------------------------------------------------------------
# Serialized rate, Eq. (5)
# --------------------------------------------------------------------------
def ceil_log2(n: int) -> int:
    return max(0, (int(n) - 1).bit_length())


def seed_bits(S: int) -> int:
    return ceil_log2(S)


def index_bits(params: Params, T_total: int) -> int:
    return params.idx_bits if params.idx_bits else ceil_log2(T_total)


def record_bytes(params: Params, T_total: int, scale_bits: Optional[int] = None) -> int:
    """L_rec = ceil((index bits + ceil(log2 S) + scale bits + P*b) / 8)   (Eq. (5)).

    The payload is ceil(log2 S) + b_e + P*b bits with b_e the scale width: 8
    for the power-of-two exponent, 16 for the fp16 scale (the parameters'
    format unless given)."""
    if scale_bits is None:
        scale_bits = params.scale_bits
    bits = index_bits(params, T_total) + seed_bits(params.S) + params.P * params.b + scale_bits
    return (bits + 7) // 8


def header_bytes(n_modules: int) -> int:
    return HEADER_FIXED_BYTES + 8 * n_modules


def budget_bytes(bpw: float, n_weights: int) -> int:
    """Byte budget of a scope-bpw target: floor(bpw * N / 8) in IEEE double."""
    return int(math.floor((bpw * n_weights) / 8.0))


def prefix_K(budget: int, h: int, L_rec: int, n_eligible: int) -> int:
    """Longest record prefix within the budget, header included (Sec. 4, Eq. (5))."""
    if budget < h:
        raise ValueError("budget smaller than the stream header")
    return min(n_eligible, (budget - h) // L_rec)


def scope_bpw(n_bytes: int, n_weights: int) -> float:
    return 8.0 * n_bytes / n_weights


# --------------------------------------------------------------------------
# Records and stream (REC-v1 / STREAM-v1)
# --------------------------------------------------------------------------
def pack_record(idx: int, seed: int, codes: Sequence[int], scale16: int,
                idx_bits: int, s_bits: int, b: int, L_rec: int, scale_bits: int = SCALE_BITS_FP16) -> bytes:
    """REC-v1: one little-endian, LSB-first bit stream holding the tile index
    (idx_bits), seed selector (ceil(log2 S) bits), P two's-complement b-bit
    coefficients and the scale field (16-bit fp16, or the 8-bit biased
    exponent), zero-padded to L_rec bytes (the fields of Sec. 3.2 in the
    widths of Eq. (5))."""
    v, pos = 0, 0
    assert 0 <= idx < (1 << idx_bits), "tile index does not fit its field"
    assert 0 <= seed < (1 << s_bits), "seed does not fit its field"
    v |= idx << pos
    pos += idx_bits
    v |= seed << pos
    pos += s_bits
    for c in codes:
        v |= (int(c) & ((1 << b) - 1)) << pos
        pos += b
    assert 0 <= int(scale16) < (1 << scale_bits), "scale does not fit its field"
    v |= int(scale16) << pos
    pos += scale_bits
    assert pos <= 8 * L_rec
    return v.to_bytes(L_rec, "little")


def unpack_record(rec: bytes, idx_bits: int, s_bits: int, P: int, b: int, scale_bits: int = SCALE_BITS_FP16):
    v = int.from_bytes(rec, "little")
    idx = v & ((1 << idx_bits) - 1)
    v >>= idx_bits
    seed = v & ((1 << s_bits) - 1)
    v >>= s_bits
    codes = []
    for _ in range(P):
        c = v & ((1 << b) - 1)
        if c >> (b - 1):
            c -= 1 << b
        codes.append(c)
        v >>= b
    scale16 = v & ((1 << scale_bits) - 1)
    return idx, seed, codes, scale16


def stream_header(params: Params, modules: Sequence[Tuple[int, int]], per_module: bool) -> bytes:
    """STREAM-v1 header: 40 fixed bytes then (rows u32, cols u32) per module.

    magic 'AWSR' | version u16 | flags u16 (bits 0-3 generator version,
    bits 4-7 scale format (0 = fp16, 1 = pow2), bit 8 per-module quotas) | C u16 | P u8 |
    b u8 | S u32 | index bits u8 | seed bits u8 | scale bits u8 | L_rec u8 |
    basis key u64 | T_total u64 | n_modules u32, all little-endian.
    """
    T_total = sum(r * c // params.C for r, c in modules)
    L = record_bytes(params, T_total)
    flags = (params.gen_version & 0xF) | ((params.scale_fmt & 0xF) << 4) | ((1 if per_module else 0) << 8)
    head = struct.pack("<4sHHHBBIBBBBQQI", MAGIC, STREAM_VERSION, flags, params.C, params.P,
                       params.b, params.S, index_bits(params, T_total), seed_bits(params.S),
                       params.scale_bits, L, params.basis_key & MASK64, T_total, len(modules))
    assert len(head) == HEADER_FIXED_BYTES
    return head + b"".join(struct.pack("<II", r, c) for r, c in modules)


def parse_header(stream: bytes):
    (magic, ver, flags, C, P, b, S, ib, sb, scb, L, key, T_total, n_mod) = struct.unpack_from(
        "<4sHHHBBIBBBBQQI", stream, 0)
    if magic != MAGIC or ver != STREAM_VERSION:
        raise ValueError("not an AWSRC stream")
    mods = [struct.unpack_from("<II", stream, HEADER_FIXED_BYTES + 8 * i) for i in range(n_mod)]
    h = header_bytes(n_mod)
    return {"flags": flags, "gen_version": flags & 0xF, "scale_fmt": (flags >> 4) & 0xF, "C": C, "P": P,
            "b": b, "S": S,
            "idx_bits": ib, "seed_bits": sb, "scale_bits": scb, "L_rec": L, "basis_key": key,
            "T_total": T_total, "modules": mods, "h": h}


def rank_order(gain: np.ndarray, tile_ids: np.ndarray) -> np.ndarray:
    """Eligible records (gain > 0) ordered by decreasing rho, ties by lower tile
    index (Eq. (4), Sec. 3.3).  With a constant L_rec, rho order = gain order."""
    elig = np.nonzero(gain > 0)[0]
    order = np.lexsort((tile_ids[elig], -gain[elig]))
    return elig[order]


def build_stream(params: Params, modules: Sequence[Tuple[int, int]], enc: Dict[str, np.ndarray],
                 bpw: float, per_module: bool) -> Tuple[bytes, int, int]:
    """Rank records and serialize the stream for one scope-bpw budget.

    enc holds the per-tile encoder outputs for all modules concatenated in
    module order (global tile index = module tile offset + local tile).
    Global mode (P variant): one ranking and the longest prefix within the
    budget, header included.  Per-module mode (U variant): module m keeps
    min(eligible_m, floor(floor(bpw*N_m/8) / L_rec)) of its best records and the
    sections follow in module order; the header is counted once, globally.
    Returns (stream bytes, K, number of eligible records).
    """
    T_total = sum(r * c // params.C for r, c in modules)
    L = record_bytes(params, T_total)
    h = header_bytes(len(modules))
    ib = index_bits(params, T_total)
    sbits = seed_bits(params.S)
    gain = np.asarray(enc["gain"])
    tile_ids = np.arange(T_total, dtype=np.int64)
    n_elig = int(np.sum(gain > 0))
    if not per_module:
        order = rank_order(gain, tile_ids)
        K = prefix_K(budget_bytes(bpw, sum(r * c for r, c in modules)), h, L, n_elig)
        chosen = order[:K]
    else:
        chosen_parts = []
        off = 0
        for r, c in modules:
            n_t = r * c // params.C
            sl = slice(off, off + n_t)
            order = rank_order(gain[sl], tile_ids[sl])
            K_m = min(len(order), budget_bytes(bpw, r * c) // L)
            chosen_parts.append(order[:K_m] + off)
            off += n_t
        chosen = np.concatenate(chosen_parts) if chosen_parts else np.zeros(0, np.int64)
        K = len(chosen)
    body = b"".join(pack_record(int(t), int(enc["seed"][t]), enc["codes"][t], int(enc["scale"][t]),
                                ib, sbits, params.b, L, params.scale_bits) for t in chosen)
    return stream_header(params, modules, per_module) + body, K, n_elig


# --------------------------------------------------------------------------
# Decoder (Sec. 3.2): regenerate B_s and add B_s alpha_hat onto W0
# --------------------------------------------------------------------------
def decode_add(stream: bytes, W0_list: Sequence[np.ndarray]) -> List[np.ndarray]:
    """Repaired weights W_hat = W0 + R_hat in float64 (Eq. (1)).

    Each record regenerates its basis from (basis key, seed) and adds
    B_s (scale * q) onto its tile; tiles without a record keep W0 unchanged,
    so an empty stream returns W0 exactly.
    """
    hd = parse_header(stream)
    C, P, b = hd["C"], hd["P"], hd["b"]
    L, h = hd["L_rec"], hd["h"]
    if (len(stream) - h) % L:
        raise ValueError("stream does not end on a record boundary")
    out = [np.asarray(w, dtype=np.float64).copy() for w in W0_list]
    offsets = np.cumsum([0] + [r * c // C for r, c in hd["modules"]])
    cache: Dict[int, np.ndarray] = {}
    for k in range((len(stream) - h) // L):
        rec = stream[h + k * L: h + (k + 1) * L]
        t, s, codes, s16 = unpack_record(rec, hd["idx_bits"], hd["seed_bits"], P, b, hd["scale_bits"])
        mi = int(np.searchsorted(offsets, t, side="right") - 1)
        r_, c_ = hd["modules"][mi]
        local = t - offsets[mi]
        row, blk = divmod(int(local), c_ // C)
        if s not in cache:
            cache[s] = basis_matrix(hd["basis_key"], s, C, P, hd["gen_version"])
        if hd["scale_fmt"] == SCALE_POW2:
            sc = math.ldexp(1.0, int(s16) - POW2_BIAS)
        else:
            sc = float(np.array([s16], dtype=np.uint16).view(np.float16)[0])
        out[mi][row, blk * C:(blk + 1) * C] += cache[s] @ (sc * np.asarray(codes, dtype=np.float64))
    return out


def weighted_error(W32: np.ndarray, What: np.ndarray, d: np.ndarray) -> float:
    """sum over all coordinates of d (W - W_hat)^2 for one module."""
    rows, cols = W32.shape
    D = np.broadcast_to(np.asarray(d, dtype=np.float64), (rows, cols))
    E = np.asarray(W32, dtype=np.float64) - What
    return float(np.sum(D * E * E))
