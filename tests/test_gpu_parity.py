"""Parity of the HIP path (through the C ABI) with the fp64 CPU oracle.

Every test feeds both sides the same seeded synthetic tensors.  Bars:
* backbone codes, scales, zero points and W0: bit-exact;
* encoder seed: equal to the oracle's, or the oracle's gain for the GPU's
  seed lies within 1e-6 (relative) of the oracle's best gain;
* where seeds agree: codes and fp16 scale bit-exact unless the oracle flags
  a coefficient within 1e-9 of a rounding midpoint; gain within 1e-10 of the
  tile's weighted energy; unquantized coefficients within 1e-4 of max |alpha*|;
* streams built from the same records: byte-identical;
* repaired weights: fp32 targets within 2^-22 relative (one fp32 rounding of
  the add), bf16 targets within one bf16 half-ulp; untouched tiles bit-identical.
"""
import numpy as np
import pytest
import torch

import oracle_pool as OP
from oracle import awsrc_oracle as O
from synth import WORKLOADS, Module, gen_module_inputs, gen_records, workload

pytestmark = pytest.mark.gpu

awsrc = pytest.importorskip("paper_2608_23144_amd")

DEV = "cuda"


def _u16(t):
    return (t.to(torch.int32) & 0xFFFF).cpu().numpy()


def _params(wl, fmt=0, gen=1, **kw):
    return awsrc.make_params(wl.C, wl.P, wl.b, wl.S, basis_key=wl.basis_key, ridge_lambda=wl.ridge_lambda,
                             idx_bits=wl.idx_bits, scale_fmt=fmt, gen_version=gen, **kw)


def _oparams(wl, fmt=0, gen=1):
    return O.Params(C=wl.C, P=wl.P, b=wl.b, S=wl.S, basis_key=wl.basis_key, ridge_lambda=wl.ridge_lambda,
                    idx_bits=wl.idx_bits, scale_fmt=fmt, gen_version=gen)


def _gpu_module(wl, m, want_alpha=True, fmt=0, gen=1):
    inp = gen_module_inputs(wl, m, DEV)
    codes, scale, zero, W0 = awsrc.awsrc_backbone_rtn(inp["W"])
    enc = awsrc.awsrc_encode_tiles(_params(wl, fmt, gen), inp["W"], W0, inp["d"], want_alpha=want_alpha)
    torch.cuda.synchronize()
    return inp, (codes, scale, zero, W0), enc


def _check_encode_sample(wl, m, inp, W0_gpu, enc, tiles_idx, fmt=0, gen=1):
    """Oracle on a subset of tiles of one module, with every seed's gain kept,
    compared with the GPU's outputs for them (bars in tests/oracle_pool.py)."""
    W32 = inp["W32"].cpu().numpy()
    d = inp["d"].cpu().numpy()
    _, _, _, W0o = O.rtn_backbone(W32)
    assert np.array_equal(W0o, W0_gpu.cpu().numpy())
    R = O.tiles(O.residual(W32, W0o), wl.C)[tiles_idx]
    D = O.tile_weights(d, m.rows, m.cols, wl.C)[tiles_idx]
    op = _oparams(wl, fmt, gen)
    out = OP.compare_encode(R, D, op, _u16(enc["seed"])[tiles_idx], enc["codes"].cpu().numpy()[tiles_idx],
                            _u16(enc["scale"])[tiles_idx], enc["gain"].cpu().numpy()[tiles_idx],
                            enc["alpha"].cpu().numpy()[tiles_idx] if enc.get("alpha") is not None else None)
    assert out["failures"] == 0, "\n".join(out["report"])
    return out["seed_diff"]


# ------------------------------------------------------------------ backbone
@pytest.mark.parametrize("group", [64, 128, 256])
@pytest.mark.parametrize("name,rows,cols", [("linear256", 256, 256), ("down3b", 130, 11008),
                                            ("block3b", 3, 2048)])
def test_backbone_bit_exact(name, rows, cols, group):
    wl = workload(name)
    m = Module("t", rows, cols, 0, 5, 5)
    W = gen_module_inputs(wl, m, DEV)["W"]
    codes, scale, zero, W0 = awsrc.awsrc_backbone_rtn(W, group=group)
    co, so, zo, W0o = O.rtn_backbone(W.to(torch.float32).cpu().numpy(), group=group)
    assert np.array_equal(codes.cpu().numpy(), co)
    assert np.array_equal(_u16(scale), so)
    assert np.array_equal(zero.cpu().numpy(), zo)
    assert np.array_equal(W0.cpu().numpy(), W0o)


def test_backbone_edge_groups():
    W = torch.randn(4, 512, dtype=torch.float32) * 0.02
    W[0, :128] = 0.5                      # degenerate group
    W[1, :128] = torch.arange(128) % 16 * 0.25 - 1.0   # exact grid
    W[2, 128:256] = 0
    W[2, 128] = 15.0
    W[2, 129] = 2.5                       # half-even tie
    W[3, 256:384] *= 1e7                  # scale saturates at 65504
    Wd = W.to(DEV)
    codes, scale, zero, W0 = awsrc.awsrc_backbone_rtn(Wd)
    co, so, zo, W0o = O.rtn_backbone(W.numpy())
    assert np.array_equal(codes.cpu().numpy(), co) and np.array_equal(_u16(scale), so)
    assert np.array_equal(zero.cpu().numpy(), zo) and np.array_equal(W0.cpu().numpy(), W0o)


# ------------------------------------------------------------------ encoder
def test_encode_linear256_full():
    """Small fp32 layer (C=64, S=64, P=4, b=4, per-column weights): every tile."""
    wl = WORKLOADS["linear256"]
    m = wl.modules[0]
    inp, bb, enc = _gpu_module(wl, m)
    nd = _check_encode_sample(wl, m, inp, bb[3], enc, np.arange(m.rows * m.cols // wl.C))
    assert nd <= 2


@pytest.mark.parametrize("C,P,b,S,rows,cols,d_mode", [
    (64, 8, 4, 32, 67, 512, "elem"),    # ragged wavefront, per-element weights
    (128, 8, 3, 24, 5, 256, "col"),
    (32, 4, 4, 16, 1, 128, "elem"),     # one row
    (16, 4, 4, 16, 9, 128, "col"),      # the paper's P_F operating point shape
    (64, 3, 5, 10, 20, 128, "col"),     # padded P
    (128, 2, 4, 2, 8, 256, "col"),      # the paper's U operating point shape
    (128, 8, 4, 64, 70, 512, "col"),    # matrix-core C=128 screen: ragged 32-row waves, seed ranges
    (128, 5, 4, 33, 40, 256, "col"),    # odd S: the last seed pair has one seed
    (64, 16, 8, 8, 4, 128, "elem"),
    # the pruned per-column screen (C = 64): odd S with ragged rows, seed
    # ranges of 16 pairs (each starting its pruning afresh), P = 1, b = 2,
    # and a single seed pair
    (64, 8, 4, 33, 70, 256, "col"),
    (64, 8, 4, 256, 130, 640, "col"),
    (64, 1, 4, 64, 64, 128, "col"),
    (64, 4, 2, 48, 65, 256, "col"),
    (64, 8, 4, 2, 10, 128, "col"),
])
def test_encode_small_shapes(C, P, b, S, rows, cols, d_mode):
    wl = workload("block3b", C=C, P=P, b=b, S=S, d_mode=d_mode)
    m = Module("t", rows, cols, 0, 2, 2)
    inp, bb, enc = _gpu_module(wl, m)
    T = rows * cols // C
    nd = _check_encode_sample(wl, m, inp, bb[3], enc, np.arange(T))
    assert nd <= max(1, T // 50)


@pytest.mark.parametrize("P,S,rows,cols,d_mode", [(8, 48, 70, 256, "col"), (3, 30, 64, 128, "col"),
                                                   (5, 62, 129, 256, "col"), (8, 40, 67, 256, "elem"),
                                                   (4, 256, 64, 128, "elem")])
def test_encode_f32_weights_one_seed_range(P, S, rows, cols, d_mode):
    """fp32 weights on the C = 64 matrix-core screens: per-column weights where
    one wavefront screens every seed of its tiles (fewer than 32 seed pairs),
    so the screen also runs the fp64 re-score; per-element weights with one
    and with several seed ranges; ragged row groups and padded P."""
    wl = workload("linear256", P=P, S=S, d_mode=d_mode)
    assert wl.w_dtype == "f32" and wl.d_mode == d_mode and wl.C == 64
    m = Module("t", rows, cols, 0, 2, 2)
    inp, bb, enc = _gpu_module(wl, m)
    T = rows * cols // wl.C
    nd = _check_encode_sample(wl, m, inp, bb[3], enc, np.arange(T))
    assert nd <= max(1, T // 50)


@pytest.mark.parametrize("C,P,b,S,rows,cols,d_mode", [
    (64, 8, 4, 32, 67, 512, "col"),     # matrix-core screen, per-column factors
    (64, 8, 4, 32, 67, 512, "elem"),    # matrix-core screen, per-element factors
    (128, 8, 3, 24, 40, 256, "col"),    # matrix-core C=128 screen
    (16, 4, 4, 16, 9, 128, "col"),      # the paper's P_F operating point shape, vector screen
    (32, 4, 4, 16, 3, 128, "elem"),     # vector screen, per-element weights
])
def test_encode_pow2_scale(C, P, b, S, rows, cols, d_mode):
    """Power-of-two scale exponent (Sec. 3.2) in every screen and the re-score."""
    wl = workload("block3b", C=C, P=P, b=b, S=S, d_mode=d_mode)
    m = Module("t", rows, cols, 0, 3, 3)
    inp, bb, enc = _gpu_module(wl, m, fmt=1)
    T = rows * cols // C
    nd = _check_encode_sample(wl, m, inp, bb[3], enc, np.arange(T), fmt=1)
    assert nd <= max(1, T // 50)
    assert int(_u16(enc["scale"]).max()) < 256


@pytest.mark.parametrize("C,P,b,S,rows,cols,d_mode", [
    (64, 8, 4, 32, 67, 512, "col"),     # matrix-core screen, factors from the permuted Gram
    (64, 8, 4, 32, 67, 512, "elem"),    # vector screen: per-seed transform of the permuted d
    (128, 8, 3, 24, 40, 256, "col"),    # matrix-core C=128 screen
    (16, 4, 4, 16, 9, 128, "col"),      # vector screen, per-column factors
    (32, 4, 4, 16, 3, 128, "elem"),
    (128, 16, 4, 8, 4, 256, "elem"),    # two sign words and two pattern words per column
])
def test_encode_generator_v2(C, P, b, S, rows, cols, d_mode):
    """Basis generator version 2 (seeded coordinate permutation, Eq. (2)) in
    every screen and the fp64 re-score."""
    wl = workload("block3b", C=C, P=P, b=b, S=S, d_mode=d_mode)
    m = Module("t", rows, cols, 0, 4, 4)
    inp, bb, enc = _gpu_module(wl, m, gen=2)
    T = rows * cols // C
    nd = _check_encode_sample(wl, m, inp, bb[3], enc, np.arange(T), gen=2)
    assert nd <= max(1, T // 50)


def test_pipeline_generator_v2_matches_oracle():
    """Version-2 encode, rank and decode against the oracle's stream: the
    records the GPU ranks are the oracle's where seeds agree, the stream's
    header names version 2, and the GPU decodes the oracle's stream."""
    wl = workload("linear256", S=16)
    m = wl.modules[0]
    inp, (codes, scale, zero, W0), enc = _gpu_module(wl, m, want_alpha=False, gen=2)
    p = _params(wl, gen=2)
    s, K, ne = awsrc.awsrc_rank_prefix(p, [(m.rows, m.cols)], awsrc.AWSRC_MODE_GLOBAL, 2.0, enc["seed"],
                                       enc["codes"], enc["scale"], enc["gain"])
    stream = bytes(s.cpu().numpy().tobytes())
    hd = O.parse_header(stream)
    assert hd["gen_version"] == 2 and K > 0
    W0n = W0.cpu().numpy()
    # the oracle decodes the GPU stream exactly as the GPU does (fp32 targets)
    want = O.decode_add(stream, [W0n])[0]
    out = W0.clone()
    awsrc.awsrc_decode_add(s, [out])
    w0f = W0n.astype(np.float64)
    assert np.all(np.abs(out.cpu().numpy() - want) <= 2.0 ** -22 * (np.abs(w0f) + np.abs(want - w0f)) + 1e-30)
    # and the decoded error drops by the GPU's gains of the listed records
    W32 = inp["W32"].cpu().numpy()
    d = inp["d"].cpu().numpy()
    Dfull = np.broadcast_to(d, W32.shape) if d.ndim == 1 else d
    e0 = O.weighted_error(W32, w0f, Dfull)
    e1 = O.weighted_error(W32, want, Dfull)
    gain = enc["gain"].cpu().numpy()
    order = O.rank_order(gain, np.arange(gain.size))[:K]
    assert abs((e0 - e1) - float(np.sum(gain[order]))) <= 1e-8 * e0


def test_encode_zero_residual_tiles():
    """Tiles whose residual is exactly zero keep seed 0, an all-zero record and gain 0."""
    wl = workload("linear256", S=8)
    W = torch.zeros(64, 256, dtype=torch.float32, device=DEV)
    W[:, 128:] = torch.randn(64, 128, device=DEV) * 0.02
    d = torch.exp(torch.randn(256, device=DEV))
    codes, scale, zero, W0 = awsrc.awsrc_backbone_rtn(W)
    enc = awsrc.awsrc_encode_tiles(_params(wl), W, W0, d)
    nb = 256 // 64
    seed = _u16(enc["seed"]).reshape(64, nb)
    gain = enc["gain"].cpu().numpy().reshape(64, nb)
    assert np.all(seed[:, :2] == 0) and np.all(gain[:, :2] == 0)
    assert np.all(enc["codes"].cpu().numpy().reshape(64, nb, -1)[:, :2] == 0)
    assert np.all(_u16(enc["scale"]).reshape(64, nb)[:, :2] == 0)


def test_encode_scored_count():
    """awsrc_encode_scored: the pruned screens (C = 64, per-column and
    per-element weights) score every tile's first seeds and, on realistic
    data, a small part of the rest.  The per-column module has enough row
    groups that each wavefront searches all S seeds (with seed ranges split
    over wavefronts, each range starts its pruning afresh); the per-element
    screen always searches all seeds per wavefront, and each lane queues up
    to four survivors before the first scoring round."""
    wl = WORKLOADS["down3b"]
    m = Module("scored", 2048, 4096, 0, 1, 1)
    inp, bb, enc = _gpu_module(wl, m)
    T, S = m.rows * m.cols // wl.C, wl.S
    sc = awsrc.awsrc_encode_scored(enc)
    assert 2 * T <= sc < T * S // 8, (sc, T * S)
    idx = np.arange(0, T, 997)
    assert _check_encode_sample(wl, m, inp, bb[3], enc, idx) <= 1
    wl2 = WORKLOADS["block3b"]
    m2 = Module("scored_pe", 256, 2048, 0, 1, 1)
    inp2, bb2, enc2 = _gpu_module(wl2, m2)
    T2 = m2.rows * m2.cols // wl2.C
    sc2 = awsrc.awsrc_encode_scored(enc2)
    assert 4 * T2 <= sc2 < T2 * wl2.S // 8, (sc2, T2 * wl2.S)
    assert _check_encode_sample(wl2, m2, inp2, bb2[3], enc2, np.arange(0, T2, 331)) <= 1


# ------------------------------------------------------------------ SDQ backbone
@pytest.mark.parametrize("name,rows,cols", [("down3b", 64, 11008), ("down3b", 2048, 11008), ("linear256", 256, 256)])
def test_sdq_backbone_bit_exact(name, rows, cols):
    """SDQ codes, block means and steps of the GPU's RTN scales, and the
    RTN-INT4-SDQ W0, bit-exact against the oracle (64 x 11008 has 5504
    groups: 21 full blocks and one of 128)."""
    wl = WORKLOADS[name]
    m = Module("sdq", rows, cols, 0, 1, 1)
    inp = gen_module_inputs(wl, m, DEV)
    codes, scale, zero, W0 = awsrc.awsrc_backbone_rtn(inp["W"])
    sdq = awsrc.awsrc_sdq_encode(scale)
    W0s = awsrc.awsrc_backbone_sdq_dequant(codes, zero, sdq)
    torch.cuda.synchronize()
    s16 = scale.cpu().numpy().view(np.uint16)
    oc, om, ost = O.sdq_encode(s16)
    assert np.array_equal(sdq[0].cpu().numpy(), oc)
    assert np.array_equal(sdq[1].cpu().numpy().view(np.uint32), om.view(np.uint32))
    assert np.array_equal(sdq[2].cpu().numpy().view(np.uint32), ost.view(np.uint32))
    want = O.rtn_dequant_sdq(codes.cpu().numpy(), zero.cpu().numpy(), oc, om, ost)
    assert np.array_equal(W0s.cpu().numpy().view(np.uint32), want.view(np.uint32))
    # SDQ moves W0 by at most half a scale step per weight unit of (q - z)
    assert (W0s - W0).abs().max().item() <= 15 * 0.5 * float(ost.max()) * (1 + 1e-6) + 1e-12


def test_sdq_constant_and_degenerate_blocks():
    """Blocks whose scales are all equal code to zero and reproduce the RTN-v1
    W0 bit for bit; an all-zero weight matrix (every group degenerate, scale
    1.0) does too."""
    for W in (torch.zeros(8, 4096, device=DEV),
              torch.linspace(-1, 1, 128, device=DEV).repeat(4, 64).contiguous()):
        codes, scale, zero, W0 = awsrc.awsrc_backbone_rtn(W)
        sdq = awsrc.awsrc_sdq_encode(scale)
        W0s = awsrc.awsrc_backbone_sdq_dequant(codes, zero, sdq)
        torch.cuda.synchronize()
        assert torch.all(sdq[0] == 0) and torch.all(sdq[2] == 0)
        assert torch.equal(W0s.view(torch.int32), W0.view(torch.int32))


# ------------------------------------------------------------------ ranking
@pytest.mark.parametrize("mode", ["global", "per_module"])
@pytest.mark.parametrize("bpw", [0.05, 0.162, 2.0, 64.0])
def test_rank_stream_byte_exact(mode, bpw):
    op = O.Params(C=64, P=8, b=4, S=256)
    p = awsrc.make_params(64, 8, 4, 256)
    mods = [(64, 512), (8, 11008), (200, 128)]
    T = sum(r * c // 64 for r, c in mods)
    rec = gen_records(T, 8, 4, 256, seed=11)
    h = O.header_bytes(len(mods))
    if mode == "global" and O.budget_bytes(bpw, sum(r * c for r, c in mods)) < h:
        pytest.skip("budget below header")
    enc = {"seed": rec["seed"].numpy().astype(np.int64) & 0xFFFF, "codes": rec["codes"].numpy().astype(np.int64),
           "scale": rec["scale"].numpy().astype(np.int64) & 0xFFFF, "gain": rec["gain"].numpy()}
    want, K_o, ne_o = O.build_stream(op, mods, enc, bpw, per_module=(mode == "per_module"))
    dev = {k: v.to(DEV) for k, v in rec.items()}
    m = awsrc.AWSRC_MODE_GLOBAL if mode == "global" else awsrc.AWSRC_MODE_PER_MODULE
    s, K, ne = awsrc.awsrc_rank_prefix(p, mods, m, bpw, dev["seed"], dev["codes"], dev["scale"], dev["gain"])
    assert (K, ne) == (K_o, ne_o)
    assert bytes(s.cpu().numpy().tobytes()) == want


def test_rank_large_segment_with_ties():
    """Many exact ties straddling the cut: equal gains keep the lower tile index."""
    op = O.Params(C=64, P=4, b=4, S=64)
    p = awsrc.make_params(64, 4, 4, 64)
    mods = [(4096, 4096)]
    T = 4096 * 64
    rec = gen_records(T, 4, 4, 64, seed=5, frac_ties=0.6)
    enc = {"seed": rec["seed"].numpy().astype(np.int64), "codes": rec["codes"].numpy().astype(np.int64),
           "scale": rec["scale"].numpy().astype(np.int64) & 0xFFFF, "gain": rec["gain"].numpy()}
    for bpw in (0.01, 0.3):
        want, K_o, _ = O.build_stream(op, mods, enc, bpw, per_module=False)
        dev = {k: v.to(DEV) for k, v in rec.items()}
        s, K, _ = awsrc.awsrc_rank_prefix(p, mods, awsrc.AWSRC_MODE_GLOBAL, bpw, dev["seed"], dev["codes"],
                                          dev["scale"], dev["gain"])
        assert K == K_o and bytes(s.cpu().numpy().tobytes()) == want


def test_rank_stack3b_scale_global_order():
    """Global ranking at the size of the 36-layer stack (252 modules, 43.35M
    tiles, 0.32 bpw: about 9.2M records): K from the budget, the records'
    tile order equal to an independent numpy ordering of the eligible tiles
    by (-gain, tile), and the packed fields of sampled records equal to the
    encoder outputs they came from."""
    wl = WORKLOADS["stack3b"]
    shapes = [(m.rows, m.cols) for m in wl.modules]
    T = wl.n_tiles
    bpw = 0.32
    rec = gen_records(T, wl.P, wl.b, wl.S, seed=77, device=DEV)
    s, K, ne = awsrc.awsrc_rank_prefix(_params(wl), shapes, awsrc.AWSRC_MODE_GLOBAL, bpw, rec["seed"],
                                       rec["codes"], rec["scale"], rec["gain"])
    gain = rec["gain"].cpu().numpy()
    L = O.record_bytes(_oparams(wl), T)
    h = O.header_bytes(len(shapes))
    N = sum(r * c for r, c in shapes)
    assert ne == int((gain > 0).sum())
    assert K == min(ne, (O.budget_bytes(bpw, N) - h) // L) and K > 1_000_000
    assert len(s) == h + K * L
    # the top K by (-gain, tile): every gain above the K-th, then the lowest
    # tiles among those equal to it, ordered with lexsort
    elig = np.nonzero(gain > 0)[0]
    g = gain[elig]
    v = -np.partition(-g, K - 1)[K - 1]
    above = elig[g > v]
    eq = elig[g == v]
    chosen = np.concatenate([above, eq[:K - len(above)]])
    want = chosen[np.lexsort((chosen, -gain[chosen]))]
    raw = s[h:].cpu().numpy().reshape(K, L)
    assert L >= 4 and wl.idx_bits == 32
    got = raw[:, :4].copy().view("<u4").ravel().astype(np.int64)
    assert np.array_equal(got, want)
    # sampled records: seed, codes and scale of the tile they name
    hd = O.parse_header(bytes(s[:h].cpu().numpy().tobytes()))
    seed = rec["seed"].cpu().numpy().astype(np.int64) & 0xFFFF
    codes = rec["codes"].cpu().numpy()
    scale = rec["scale"].cpu().numpy().astype(np.int64) & 0xFFFF
    for k in np.random.default_rng(3).integers(0, K, 2000):
        t, sd, cd, sc = O.unpack_record(bytes(raw[k]), hd["idx_bits"], hd["seed_bits"], hd["P"], hd["b"],
                                        hd["scale_bits"])
        assert t == want[k] and sd == seed[t] and sc == scale[t] and list(cd) == codes[t].tolist()
    del rec, s
    torch.cuda.empty_cache()


def test_rank_stream_capacity_too_small():
    """K is found on the device; a stream buffer too small for the records is
    reported as AWSRC_ENOSPC after the fact, with nothing written past it."""
    p = awsrc.make_params(64, 4, 4, 64)
    mods = [(64, 1024)]
    rec = gen_records(1024, 4, 4, 64, seed=3, frac_nonpositive=0.0)
    dev = {k: v.to(DEV) for k, v in rec.items()}
    h = O.header_bytes(1)
    L = O.record_bytes(O.Params(C=64, P=4, b=4, S=64), 1024)
    buf = torch.full((h + 3 * L + 64,), 0xAB, dtype=torch.uint8, device=DEV)
    with pytest.raises(awsrc.AwsrcError) as ei:
        awsrc.awsrc_rank_prefix(p, mods, awsrc.AWSRC_MODE_GLOBAL, 8.0, dev["seed"], dev["codes"], dev["scale"],
                                dev["gain"], stream_cap=h + 3 * L, out=buf)
    assert ei.value.status == awsrc.AWSRC_ENOSPC
    assert torch.all(buf[h + 3 * L:].cpu() == 0xAB)


def test_rank_no_eligible_records():
    p = awsrc.make_params(64, 4, 4, 64)
    rec = gen_records(64, 4, 4, 64, seed=1)
    gain = -torch.abs(rec["gain"]).to(DEV)
    s, K, ne = awsrc.awsrc_rank_prefix(p, [(16, 256)], awsrc.AWSRC_MODE_GLOBAL, 8.0, rec["seed"].to(DEV),
                                       rec["codes"].to(DEV), rec["scale"].to(DEV), gain)
    assert K == 0 and ne == 0 and s.numel() == O.header_bytes(1)


# ------------------------------------------------------------------ decoding
def _oracle_stream(C, P, b, S, mods, bpw, seed, key=0):
    op = O.Params(C=C, P=P, b=b, S=S, basis_key=key)
    T = sum(r * c // C for r, c in mods)
    rec = gen_records(T, P, b, S, seed=seed)
    enc = {"seed": rec["seed"].numpy().astype(np.int64) & 0xFFFF, "codes": rec["codes"].numpy().astype(np.int64),
           "scale": rec["scale"].numpy().astype(np.int64) & 0xFFFF, "gain": rec["gain"].numpy()}
    stream, K, _ = O.build_stream(op, mods, enc, bpw, per_module=False)
    return stream, K, enc


@pytest.mark.parametrize("C,P,b,S,dtype", [(64, 8, 4, 256, torch.float32), (64, 4, 4, 64, torch.bfloat16),
                                           (128, 8, 3, 1024, torch.float32), (16, 4, 4, 16, torch.float32),
                                           (32, 16, 8, 7, torch.bfloat16)])
def test_decode_matches_oracle(C, P, b, S, dtype):
    mods = [(33, 512), (8, 1024)]
    stream, K, enc = _oracle_stream(C, P, b, S, mods, 2.0, seed=3, key=0x1234)
    g = torch.Generator().manual_seed(9)
    W0s = [(torch.randn(r, c, generator=g) * 0.02).to(dtype) for r, c in mods]
    want = O.decode_add(stream, [w.to(torch.float32).numpy() for w in W0s])
    dev = [w.to(DEV) for w in W0s]
    sb = torch.tensor(list(stream), dtype=torch.uint8, device=DEV)
    awsrc.awsrc_decode_add(sb, dev)
    hd = O.parse_header(stream)
    touched = [np.zeros((r, c // C), bool) for r, c in mods]
    offs = np.cumsum([0] + [r * c // C for r, c in mods])
    L = hd["L_rec"]
    for k in range(K):
        t = O.unpack_record(stream[hd["h"] + k * L: hd["h"] + (k + 1) * L], hd["idx_bits"], hd["seed_bits"], P, b)[0]
        mi = int(np.searchsorted(offs, t, side="right") - 1)
        rr, bb = divmod(int(t - offs[mi]), mods[mi][1] // C)
        touched[mi][rr, bb] = True
    for w0, got, ref, tm, (r, c) in zip(W0s, dev, want, touched, mods):
        got = got.to(torch.float32).cpu().numpy()
        mask = np.repeat(tm, C, axis=1)
        assert np.array_equal(got[~mask], w0.to(torch.float32).numpy()[~mask])
        tol = 2.0 ** -22 if dtype == torch.float32 else 2.0 ** -8
        w0f = w0.to(torch.float32).numpy().astype(np.float64)
        mag = np.abs(w0f) + np.abs(ref - w0f)     # operands of the add
        assert np.all(np.abs(got - ref)[mask] <= tol * mag[mask] + 1e-30)


def test_decode_many_modules():
    """More modules than the kernel stages in LDS: the module lookup reads the
    tables from global memory instead."""
    C, P, b, S = 16, 4, 4, 16
    mods = [(1 + (m % 3), 64) for m in range(300)]
    stream, K, enc = _oracle_stream(C, P, b, S, mods, 8.0, seed=21)
    assert K > 100
    g = torch.Generator().manual_seed(4)
    W0s = [torch.randn(r, c, generator=g) * 0.02 for r, c in mods]
    want = O.decode_add(stream, [w.numpy() for w in W0s])
    dev = [w.to(DEV) for w in W0s]
    awsrc.awsrc_decode_add(torch.tensor(list(stream), dtype=torch.uint8, device=DEV), dev)
    for w0, got, ref in zip(W0s, dev, want):
        got = got.cpu().numpy()
        w0f = w0.numpy().astype(np.float64)
        assert np.all(np.abs(got - ref) <= 2.0 ** -22 * (np.abs(w0f) + np.abs(ref - w0f)) + 1e-30)


def test_decode_prefixes_and_empty_stream():
    C, P, b, S = 64, 8, 4, 256
    mods = [(64, 1024)]
    stream, K, enc = _oracle_stream(C, P, b, S, mods, 4.0, seed=4)
    hd = O.parse_header(stream)
    g = torch.Generator().manual_seed(2)
    W0 = torch.randn(64, 1024, generator=g) * 0.02
    for k in (0, 1, K // 3, K):
        pre = stream[:hd["h"] + k * hd["L_rec"]]
        want = O.decode_add(pre, [W0.numpy()])[0]
        dev = W0.to(DEV)
        awsrc.awsrc_decode_add(torch.tensor(list(pre), dtype=torch.uint8, device=DEV), [dev])
        got = dev.cpu().numpy()
        if k == 0:
            assert np.array_equal(got, W0.numpy())
        w0f = W0.numpy().astype(np.float64)
        assert np.all(np.abs(got - want) <= 2.0 ** -22 * (np.abs(w0f) + np.abs(want - w0f)) + 1e-30)


def test_decode_prepare_reuses_workspace():
    """A workspace handed back to prepare is used when large enough (same
    tensor returned) and replaced when too small; results match the oracle."""
    C, P, b, S = 64, 8, 4, 256
    mods = [(64, 1024)]
    stream, K, enc = _oracle_stream(C, P, b, S, mods, 4.0, seed=6)
    hd = O.parse_header(stream)
    g = torch.Generator().manual_seed(5)
    W0 = torch.randn(64, 1024, generator=g) * 0.02
    ws = None
    for k, expect_same in ((K // 2, False), (K // 4, True), (K, False)):
        pre = stream[:hd["h"] + k * hd["L_rec"]]
        dev = W0.to(DEV)
        plan, ws2 = awsrc.awsrc_decode_prepare(torch.tensor(list(pre), dtype=torch.uint8, device=DEV), [dev],
                                               workspace=ws)
        assert (ws2 is ws) == expect_same
        awsrc.awsrc_decode_apply(plan)
        torch.cuda.synchronize()
        ws = ws2
        want = O.decode_add(pre, [W0.numpy()])[0]
        w0f = W0.numpy().astype(np.float64)
        assert np.all(np.abs(dev.cpu().numpy() - want) <= 2.0 ** -22 * (np.abs(w0f) + np.abs(want - w0f)) + 1e-30)


def _corrupt_cases(stream, hd):
    h, L = hd["h"], hd["L_rec"]
    bad = {}
    b = bytearray(stream); b[0] = ord("X"); bad["magic"] = bytes(b)
    bad["truncated"] = stream[:-1]
    b = bytearray(stream); b[h:h + L] = stream[h + L:h + 2 * L]; bad["duplicate_tile"] = bytes(b)
    b = bytearray(stream); b[h:h + 4] = (hd["T_total"] + 5).to_bytes(4, "little"); bad["tile_out_of_range"] = bytes(b)
    b = bytearray(stream); b[h + L - 1] |= 0x7C; bad["inf_scale"] = bytes(b)
    b = bytearray(stream); b[12:16] = (3).to_bytes(4, "little"); bad["header_S"] = bytes(b)
    return bad


def test_decode_rejects_corrupt_streams():
    C, P, b, S = 64, 8, 4, 256
    mods = [(32, 512)]
    stream, K, enc = _oracle_stream(C, P, b, S, mods, 4.0, seed=8)
    assert K >= 2
    hd = O.parse_header(stream)
    W0 = torch.randn(32, 512) * 0.02
    for name, bs in _corrupt_cases(stream, hd).items():
        dev = W0.to(DEV)
        with pytest.raises(awsrc.AwsrcError) as ei:
            awsrc.awsrc_decode_add(torch.tensor(list(bs), dtype=torch.uint8, device=DEV), [dev])
        assert ei.value.status == awsrc.AWSRC_ECORRUPT, name
        assert torch.equal(dev.cpu(), W0), name


# ------------------------------------------------------------------ end to end
def test_pipeline_linear256_matches_oracle():
    """backbone -> encode -> rank (0.162 bpw) -> decode on the GPU, against the
    same chain in the oracle: identical stream bytes and repaired weights."""
    wl = WORKLOADS["linear256"]
    m = wl.modules[0]
    inp, (codes, scale, zero, W0), enc = _gpu_module(wl, m)
    p = _params(wl)
    s, K, ne = awsrc.awsrc_rank_prefix(p, [(m.rows, m.cols)], awsrc.AWSRC_MODE_GLOBAL, 0.162, enc["seed"],
                                       enc["codes"], enc["scale"], enc["gain"])
    W32 = inp["W32"].cpu().numpy()
    d = inp["d"].cpu().numpy()
    _, _, _, W0o = O.rtn_backbone(W32)
    R = O.residual(W32, W0o)
    op = _oparams(wl)
    orc = O.encode_tiles(O.tiles(R, wl.C), O.tile_weights(d, m.rows, m.cols, wl.C), op)
    want, K_o, ne_o = O.build_stream(op, [(m.rows, m.cols)], orc, 0.162, per_module=False)
    assert (K, ne) == (K_o, ne_o)
    assert bytes(s.cpu().numpy().tobytes()) == want
    What = W0.clone()
    awsrc.awsrc_decode_add(s, [What])
    ref = O.decode_add(want, [W0o])[0]
    w0f = W0o.astype(np.float64)
    assert np.all(np.abs(What.cpu().numpy() - ref) <= 2.0 ** -22 * (np.abs(w0f) + np.abs(ref - w0f)) + 1e-30)
    # the repair lowers the weighted error by exactly the retained gains
    e0 = O.weighted_error(W32, W0o.astype(np.float64), d)
    e1 = O.weighted_error(W32, What.cpu().numpy().astype(np.float64), d)
    kept = np.sort(orc["gain"][orc["gain"] > 0])[::-1][:K]
    assert abs((e0 - e1) - kept.sum()) <= 1e-5 * e0


def test_pipeline_on_sdq_backbone_matches_oracle():
    """The residual codec repairing the RTN-INT4-SDQ backbone (the paper's
    Sec. 4 setting): backbone -> SDQ -> encode -> rank -> decode on the GPU
    against the same chain in the oracle: identical stream bytes and repaired
    weights."""
    wl = WORKLOADS["linear256"]
    m = wl.modules[0]
    inp = gen_module_inputs(wl, m, DEV)
    codes, scale, zero, _ = awsrc.awsrc_backbone_rtn(inp["W"])
    W0 = awsrc.awsrc_backbone_sdq_dequant(codes, zero, awsrc.awsrc_sdq_encode(scale))
    p = _params(wl)
    enc = awsrc.awsrc_encode_tiles(p, inp["W"], W0, inp["d"])
    s, K, ne = awsrc.awsrc_rank_prefix(p, [(m.rows, m.cols)], awsrc.AWSRC_MODE_GLOBAL, 0.162, enc["seed"],
                                       enc["codes"], enc["scale"], enc["gain"])
    W32 = inp["W32"].cpu().numpy()
    d = inp["d"].cpu().numpy()
    oc, _, oz, _ = O.rtn_backbone(W32)
    s16 = O.rtn_backbone(W32)[1]
    W0o = O.rtn_dequant_sdq(oc, oz, *O.sdq_encode(s16))
    assert np.array_equal(W0.cpu().numpy(), W0o)
    op = _oparams(wl)
    orc = O.encode_tiles(O.tiles(O.residual(W32, W0o), wl.C), O.tile_weights(d, m.rows, m.cols, wl.C), op)
    want, K_o, ne_o = O.build_stream(op, [(m.rows, m.cols)], orc, 0.162, per_module=False)
    assert (K, ne) == (K_o, ne_o)
    assert bytes(s.cpu().numpy().tobytes()) == want
    What = W0.clone()
    awsrc.awsrc_decode_add(s, [What])
    ref = O.decode_add(want, [W0o])[0]
    w0f = W0o.astype(np.float64)
    assert np.all(np.abs(What.cpu().numpy() - ref) <= 2.0 ** -22 * (np.abs(w0f) + np.abs(ref - w0f)) + 1e-30)


def test_pipeline_paper_pf_operating_point_pow2():
    """The paper's P_F record: (C, P, b, S) = (16, 4, 4, 16), ceil(log2 T)-bit
    index and an 8-bit power-of-two exponent; per-element weights, global
    ranking.  backbone -> encode -> rank -> decode on the GPU against the same
    chain in the oracle: identical stream bytes and repaired weights."""
    wl = workload("block3b", C=16, P=4, b=4, S=16, d_mode="elem", idx_bits=0)
    m = Module("t", 48, 256, 0, 4, 4)
    inp, (codes, scale, zero, W0), enc = _gpu_module(wl, m, fmt=1)
    p = _params(wl, 1)
    s, K, ne = awsrc.awsrc_rank_prefix(p, [(m.rows, m.cols)], awsrc.AWSRC_MODE_GLOBAL, 1.5, enc["seed"],
                                       enc["codes"], enc["scale"], enc["gain"])
    W32 = inp["W32"].cpu().numpy()
    d = inp["d"].cpu().numpy()
    _, _, _, W0o = O.rtn_backbone(W32)
    op = _oparams(wl, 1)
    orc = O.encode_tiles(O.tiles(O.residual(W32, W0o), wl.C), O.tile_weights(d, m.rows, m.cols, wl.C), op)
    want, K_o, ne_o = O.build_stream(op, [(m.rows, m.cols)], orc, 1.5, per_module=False)
    hd = O.parse_header(want)
    assert hd["L_rec"] == (10 + 4 + 16 + 8 + 7) // 8 and hd["scale_bits"] == 8 and hd["scale_fmt"] == 1
    assert (K, ne) == (K_o, ne_o) and K > 0
    assert bytes(s.cpu().numpy().tobytes()) == want
    What = W0.clone()
    awsrc.awsrc_decode_add(s, [What])
    ref = O.decode_add(want, [W0o])[0]
    w0f = W0o.astype(np.float64)
    assert np.all(np.abs(What.cpu().numpy() - ref) <= 2.0 ** -22 * (np.abs(w0f) + np.abs(ref - w0f)) + 1e-30)


def test_rank_and_decode_pow2_records():
    """Random records in the power-of-two format: byte-identical stream, and
    decoding onto bf16 and fp32 targets within the stated tolerances."""
    op = O.Params(C=64, P=8, b=4, S=256, scale_fmt=1)
    p = awsrc.make_params(64, 8, 4, 256, scale_fmt=1)
    mods = [(16, 512), (8, 1024)]
    T = sum(r * c // 64 for r, c in mods)
    rec = gen_records(T, 8, 4, 256, seed=17)
    # exponents e in [-28, 3] (fields 100..131) and some field-0 records: 2^-128
    # is a valid (subnormal) scale whose correction is negligible
    rec["scale"] = (100 + (rec["scale"].to(torch.int32) & 0x1F)).to(torch.int16)
    rec["scale"][::7] = 0
    enc = {"seed": rec["seed"].numpy().astype(np.int64) & 0xFFFF, "codes": rec["codes"].numpy().astype(np.int64),
           "scale": rec["scale"].numpy().astype(np.int64) & 0xFFFF, "gain": rec["gain"].numpy()}
    want, K_o, ne_o = O.build_stream(op, mods, enc, 4.0, per_module=False)
    dev = {k: v.to(DEV) for k, v in rec.items()}
    s, K, ne = awsrc.awsrc_rank_prefix(p, mods, awsrc.AWSRC_MODE_GLOBAL, 4.0, dev["seed"], dev["codes"],
                                       dev["scale"], dev["gain"])
    assert (K, ne) == (K_o, ne_o) and bytes(s.cpu().numpy().tobytes()) == want
    g = torch.Generator().manual_seed(3)
    for dtype, tol in ((torch.float32, 2.0 ** -22), (torch.bfloat16, 2.0 ** -8)):
        W0s = [(torch.randn(r, c, generator=g) * 0.02).to(dtype) for r, c in mods]
        refs = O.decode_add(want, [w.to(torch.float32).numpy() for w in W0s])
        outs = [w.to(DEV) for w in W0s]
        awsrc.awsrc_decode_add(s, outs)
        for w0, got, ref in zip(W0s, outs, refs):
            w0f = w0.to(torch.float32).numpy().astype(np.float64)
            diff = np.abs(got.to(torch.float32).cpu().numpy() - ref)
            assert np.all(diff <= tol * (np.abs(w0f) + np.abs(ref - w0f)) + 1e-30)


def test_pipeline_down3b_properties():
    """Full-size 3B down projection, per-module quota (U variant): stream
    structure holds at size and decoding removes exactly the retained gains."""
    wl = WORKLOADS["down3b"]
    m = wl.modules[0]
    inp, (codes, scale, zero, W0), enc = _gpu_module(wl, m, want_alpha=False)
    p = _params(wl)
    s, K, ne = awsrc.awsrc_rank_prefix(p, [(m.rows, m.cols)], awsrc.AWSRC_MODE_PER_MODULE, 0.162, enc["seed"],
                                       enc["codes"], enc["scale"], enc["gain"])
    gain = enc["gain"].cpu().numpy()
    L = O.record_bytes(_oparams(wl), gain.size)
    assert ne == int((gain > 0).sum())
    assert K == min(ne, O.budget_bytes(0.162, m.rows * m.cols) // L)
    hd = O.parse_header(bytes(s[:O.header_bytes(1)].cpu().numpy().tobytes()))
    assert hd["L_rec"] == L == 11 and len(s) == hd["h"] + K * L
    order = O.rank_order(gain, np.arange(gain.size))[:K]
    raw = s[hd["h"]:].cpu().numpy().reshape(K, L)
    idx = raw[:, :4].copy().view("<u4").ravel()
    assert np.array_equal(idx, order)
    # weighted error drop equals the sum of retained gains (fp64 on the GPU)
    What = W0.clone()
    awsrc.awsrc_decode_add(s, [What])
    W = inp["W32"].double()
    dd = inp["d"].double()[None, :]
    e0 = (dd * (W - W0.double()) ** 2).sum().item()
    e1 = (dd * (W - What.double()) ** 2).sum().item()
    assert abs((e0 - e1) - gain[order].sum()) <= 1e-6 * e0


def _reconstruct_case(C, P, b, S, mods, group, bpw, seed, fmt=0):
    """Oracle stream from seeded records, oracle backbones from seeded W; the
    GPU reconstructs into bf16 buffers pre-filled with NaN patterns."""
    op = O.Params(C=C, P=P, b=b, S=S, basis_key=0x51, scale_fmt=fmt)
    T = sum(r * c // C for r, c in mods)
    rec = gen_records(T, P, b, S, seed=seed)
    if fmt == O.SCALE_POW2:
        rec["scale"] = (100 + (rec["scale"].to(torch.int32) & 0x1F)).to(torch.int16)
    enc = {"seed": rec["seed"].numpy().astype(np.int64) & 0xFFFF, "codes": rec["codes"].numpy().astype(np.int64),
           "scale": rec["scale"].numpy().astype(np.int64) & 0xFFFF, "gain": rec["gain"].numpy()}
    stream, K, _ = O.build_stream(op, mods, enc, bpw, per_module=False)
    g = torch.Generator().manual_seed(seed + 1)
    bbs = [O.rtn_backbone((torch.randn(r, c, generator=g) * 0.02).numpy(), group)[:3] for r, c in mods]
    want = O.reconstruct_bf16(stream, bbs, group)
    W0s = [O.rtn_dequant(cd, s16, z, group) for cd, s16, z in bbs]
    dev_bb = [tuple(torch.from_numpy(np.ascontiguousarray(a)).to(DEV) for a in (cd, s16.view(np.int16), z))
              for cd, s16, z in bbs]
    outs = [torch.full((r, c), -1, dtype=torch.int16, device=DEV).view(torch.bfloat16) for r, c in mods]
    sb = torch.tensor(list(stream), dtype=torch.uint8, device=DEV)
    plan, ws = awsrc.awsrc_decode_prepare(sb, outs)
    awsrc.awsrc_reconstruct_bf16(plan, dev_bb, group)
    torch.cuda.synchronize()
    return stream, K, W0s, want, outs


def _check_reconstruct(C, stream, K, W0s, want, outs, mods):
    hd = O.parse_header(stream)
    offs = np.cumsum([0] + [r * c // C for r, c in mods])
    touched = [np.zeros((r, c // C), bool) for r, c in mods]
    L = hd["L_rec"]
    for k in range(K):
        t = O.unpack_record(stream[hd["h"] + k * L: hd["h"] + (k + 1) * L], hd["idx_bits"], hd["seed_bits"],
                            hd["P"], hd["b"], hd["scale_bits"])[0]
        mi = int(np.searchsorted(offs, t, side="right") - 1)
        rr, bk = divmod(int(t - offs[mi]), mods[mi][1] // C)
        touched[mi][rr, bk] = True
    n_exact = n_rec = 0
    for w0, got, ref, ex, tm in zip(W0s, outs, want, O.decode_add(stream, W0s), touched):
        got = got.to(torch.float32).cpu().numpy().astype(np.float64)
        mask = np.repeat(tm, C, axis=1)
        # tiles without a record: bf16(W0), one rounding of the same fp32 value
        assert np.array_equal(got[~mask], ref[~mask])
        # record tiles: both sides round to bf16 once, from sums that differ by
        # the fp32 add's rounding, so they agree to one bf16 ulp.  The oracle's
        # fp64 correction carries its own rounding of P terms, each at most the
        # tile's largest |rhat| (B_s has orthonormal columns): where the exact
        # sum is zero (W0 = 0 and the integer sum cancels) the kernel returns 0
        # and the oracle a residue below 2^-40 of that.
        w0f = w0.astype(np.float64)
        rh = np.abs(ex - w0f)
        tile_max = np.repeat(rh.reshape(rh.shape[0], -1, C).max(axis=2), C, axis=1)
        mag = np.abs(w0f) + rh
        diff = np.abs(got - ref)
        assert np.all(diff[mask] <= 2.0 ** -7 * np.abs(ref[mask]) + 2.0 ** -21 * mag[mask]
                      + 2.0 ** -40 * tile_max[mask])
        n_exact += int(np.count_nonzero(diff[mask] == 0))
        n_rec += int(np.count_nonzero(mask))
    assert n_rec == K * C
    assert n_exact >= 0.98 * n_rec


@pytest.mark.parametrize("C,P,b,S,group,mods,fmt", [
    (64, 8, 4, 256, 128, [(33, 512), (8, 1024)], 0),
    (64, 8, 4, 256, 128, [(33, 512), (8, 1024)], 1),
    (16, 4, 4, 16, 64, [(5, 128), (3, 256), (1, 64)], 0),
    (32, 5, 3, 32, 256, [(7, 256), (4, 768)], 0),
    (128, 8, 4, 64, 256, [(9, 512)], 1),
    (128, 16, 4, 64, 128, [(6, 1024)], 0),
])
def test_reconstruct_bf16_matches_oracle(C, P, b, S, group, mods, fmt):
    stream, K, W0s, want, outs = _reconstruct_case(C, P, b, S, mods, group, 2.0, seed=5, fmt=fmt)
    assert K > 0
    _check_reconstruct(C, stream, K, W0s, want, outs, mods)


@pytest.mark.parametrize("C,P,b,S,group,mods,fmt", [
    (64, 8, 4, 256, 128, [(33, 512), (8, 1024), (1, 128)], 0),
    (128, 8, 3, 64, 128, [(9, 512)], 1),
    (16, 4, 4, 16, 64, [(5, 128), (3, 256)], 0),
])
def test_reconstruct_bf16_prefixes_match_single_calls_and_oracle(C, P, b, S, group, mods, fmt):
    """Nested prefixes of one stream reconstructed in one call (five targets:
    a pass of four and a pass of one at C >= 64, single passes below; record
    counts in no particular order, an empty prefix and the whole stream among
    them) equal, bit for bit, one awsrc_reconstruct_bf16 of each prefix's own
    stream, and the oracle's reconstruction of each prefix."""
    stream, K, W0s, want_full, outs_full = _reconstruct_case(C, P, b, S, mods, group, 2.0, seed=9, fmt=fmt)
    assert K > 8
    hd = O.parse_header(stream)
    h, L = hd["h"], hd["L_rec"]
    Ks = [K // 3, 0, K, K // 2, K - 1]
    g = torch.Generator().manual_seed(10)
    bbs = [O.rtn_backbone((torch.randn(r, c, generator=g) * 0.02).numpy(), group)[:3] for r, c in mods]
    dev_bb = [tuple(torch.from_numpy(np.ascontiguousarray(a)).to(DEV) for a in (cd, s16.view(np.int16), z))
              for cd, s16, z in bbs]
    sb = torch.tensor(list(stream), dtype=torch.uint8, device=DEV)
    dummy = [torch.empty(r, c, dtype=torch.bfloat16, device=DEV) for r, c in mods]
    plan, ws = awsrc.awsrc_decode_prepare(sb, dummy)
    outs = [[torch.full((r, c), -1, dtype=torch.int16, device=DEV).view(torch.bfloat16) for r, c in mods]
            for _ in Ks]
    awsrc.awsrc_reconstruct_bf16_prefixes(plan, Ks, outs, dev_bb, group)
    torch.cuda.synchronize()
    W0o = [O.rtn_dequant(cd, s16, z, group) for cd, s16, z in bbs]
    for k, got in zip(Ks, outs):
        sub = stream[:h + k * L]
        single = [torch.full((r, c), -1, dtype=torch.int16, device=DEV).view(torch.bfloat16) for r, c in mods]
        p1, _ = awsrc.awsrc_decode_prepare(torch.tensor(list(sub), dtype=torch.uint8, device=DEV), single)
        awsrc.awsrc_reconstruct_bf16(p1, dev_bb, group)
        torch.cuda.synchronize()
        for a, c in zip(got, single):
            assert torch.equal(a.view(torch.int16), c.view(torch.int16)), k
        _check_reconstruct(C, sub, k, W0o, O.reconstruct_bf16(sub, bbs, group), got, mods)


@pytest.mark.parametrize("C,P,b,S,group,mods,fmt", [
    (64, 8, 4, 256, 128, [(33, 512), (300, 1024), (1, 128)], 0),   # ten SDQ blocks, a partial last one
    (16, 4, 4, 16, 64, [(5, 128), (3, 256)], 0),
    (64, 4, 4, 32, 128, [(2 + m % 3, 128 * (1 + m % 2)) for m in range(230)], 1),  # two module windows
])
def test_reconstruct_bf16_sdq_matches_oracle(C, P, b, S, group, mods, fmt):
    """Dense bf16 reconstruction on the RTN-INT4-SDQ backbone: into the plan's
    own targets (every record) and into four nested prefixes in one call,
    against the oracle's SDQ reconstruction of each prefix."""
    op = O.Params(C=C, P=P, b=b, S=S, basis_key=0x51, scale_fmt=fmt)
    T = sum(r * c // C for r, c in mods)
    rec = gen_records(T, P, b, S, seed=21)
    if fmt == O.SCALE_POW2:
        rec["scale"] = (100 + (rec["scale"].to(torch.int32) & 0x1F)).to(torch.int16)
    enc = {"seed": rec["seed"].numpy().astype(np.int64) & 0xFFFF, "codes": rec["codes"].numpy().astype(np.int64),
           "scale": rec["scale"].numpy().astype(np.int64) & 0xFFFF, "gain": rec["gain"].numpy()}
    stream, K, _ = O.build_stream(op, mods, enc, 2.0, per_module=False)
    assert K > 8
    g = torch.Generator().manual_seed(22)
    bbs = []
    for r, c in mods:
        cd, s16, z, _ = O.rtn_backbone((torch.randn(r, c, generator=g) * 0.02).numpy(), group)
        sc, mu, st = O.sdq_encode(s16)
        bbs.append((cd, z, sc, mu, st))
    dev_bb = [tuple(torch.from_numpy(np.ascontiguousarray(a)).to(DEV) for a in bb) for bb in bbs]
    W0s = [O.rtn_dequant_sdq(cd, z, sc, mu, st, group) for cd, z, sc, mu, st in bbs]
    sb = torch.tensor(list(stream), dtype=torch.uint8, device=DEV)
    outs = [torch.full((r, c), -1, dtype=torch.int16, device=DEV).view(torch.bfloat16) for r, c in mods]
    plan, ws = awsrc.awsrc_decode_prepare(sb, outs)
    awsrc.awsrc_reconstruct_bf16_sdq(plan, dev_bb, group=group)
    torch.cuda.synchronize()
    _check_reconstruct(C, stream, K, W0s, O.reconstruct_bf16_sdq(stream, bbs, group), outs, mods)
    hd = O.parse_header(stream)
    h, L = hd["h"], hd["L_rec"]
    Ks = [K // 3, 0, K, K // 2]
    pre = [[torch.full((r, c), -1, dtype=torch.int16, device=DEV).view(torch.bfloat16) for r, c in mods] for _ in Ks]
    awsrc.awsrc_reconstruct_bf16_sdq(plan, dev_bb, K_out=Ks, outs=pre, group=group)
    torch.cuda.synchronize()
    for k, got in zip(Ks, pre):
        sub = stream[:h + k * L]
        _check_reconstruct(C, sub, k, W0s, O.reconstruct_bf16_sdq(sub, bbs, group), got, mods)


def test_reconstruct_bf16_empty_stream_and_many_modules():
    """K = 0 gives bf16(W0) everywhere; 300 modules exceed the module table
    the dense pass stages in LDS."""
    C, P, b, S = 16, 4, 4, 16
    stream, K, W0s, want, outs = _reconstruct_case(C, P, b, S, [(8, 256)], 64, 0.19, seed=2)  # header only
    assert K == 0
    _check_reconstruct(C, stream, K, W0s, want, outs, [(8, 256)])
    mods = [(1 + (m % 3), 64 * (1 + m % 2)) for m in range(300)]
    stream, K, W0s, want, outs = _reconstruct_case(C, P, b, S, mods, 64, 6.0, seed=8)
    assert K > 100
    _check_reconstruct(C, stream, K, W0s, want, outs, mods)


def test_reconstruct_bf16_down3b_pipeline():
    """Full-size 3B down projection: GPU backbone, encoder and ranked stream,
    reconstructed in bf16; matches the oracle's reconstruction of the same
    stream and backbone, and equals decode_add onto a bf16 copy of W0 except
    where that rounds twice."""
    wl = WORKLOADS["down3b"]
    m = wl.modules[0]
    inp, (codes, scale, zero, W0), enc = _gpu_module(wl, m, want_alpha=False)
    p = _params(wl)
    s, K, ne = awsrc.awsrc_rank_prefix(p, [(m.rows, m.cols)], awsrc.AWSRC_MODE_GLOBAL, 0.162, enc["seed"],
                                       enc["codes"], enc["scale"], enc["gain"])
    assert K > 1000
    out = torch.empty(m.rows, m.cols, dtype=torch.bfloat16, device=DEV)
    plan, ws = awsrc.awsrc_decode_prepare(s, [out])
    awsrc.awsrc_reconstruct_bf16(plan, [(codes, scale, zero)], 128)
    torch.cuda.synchronize()
    stream = bytes(s.cpu().numpy().tobytes())
    # the oracle's own backbone (equal to the GPU's, bit for bit)
    bb = O.rtn_backbone(inp["W32"].cpu().numpy())[:3]
    assert np.array_equal(bb[0], codes.cpu().numpy()) and np.array_equal(bb[1], _u16(scale))
    assert np.array_equal(bb[2], zero.cpu().numpy())
    want = O.reconstruct_bf16(stream, [bb], 128)
    W0s = [O.rtn_dequant(*bb, 128)]
    assert np.array_equal(W0s[0], W0.cpu().numpy())
    _check_reconstruct(wl.C, stream, K, W0s, want, [out], [(m.rows, m.cols)])


# ------------------------------------------------------------------ batched encode
@pytest.mark.parametrize("name", ["block3b", "down3b"])
def test_encode_modules_matches_per_module_calls_and_oracle(name):
    """awsrc_encode_modules over modules of different shapes (one of them
    empty, one a single row) gives, in module order, exactly what one
    awsrc_encode_tiles call per module gives, and every tile agrees with the
    oracle (per-element weights: one batched launch; per-column weights:
    the modules one after another)."""
    wl = workload(name, S=40)
    mods = [Module("a", 70, 512, 0, 1, 1), Module("empty", 0, 256, 0, 2, 2), Module("c", 33, 1024, 0, 3, 3),
            Module("row", 1, 128, 0, 4, 4)]
    p = _params(wl)
    inps, W0s = [], []
    for m in mods:
        inp = gen_module_inputs(wl, m, DEV)
        W0s.append(awsrc.awsrc_backbone_rtn(inp["W"])[3] if m.rows else
                   torch.empty(0, m.cols, dtype=torch.float32, device=DEV))
        inps.append(inp)
    got = awsrc.awsrc_encode_modules(p, [i["W"] for i in inps], W0s, [i["d"] for i in inps], want_alpha=True)
    torch.cuda.synchronize()
    off = 0
    for m, inp, W0 in zip(mods, inps, W0s):
        T = m.rows * m.cols // wl.C
        if T == 0:
            continue
        ref = awsrc.awsrc_encode_tiles(p, inp["W"], W0, inp["d"], want_alpha=True)
        torch.cuda.synchronize()
        for k in ("seed", "codes", "scale", "alpha"):
            assert torch.equal(got[k][off:off + T], ref[k]), (m.name, k)
        assert torch.equal(got["gain"][off:off + T].view(torch.int64), ref["gain"].view(torch.int64)), m.name
        sl = {k: (v[off:off + T] if v is not None and k != "workspace" else v) for k, v in got.items()}
        _check_encode_sample(wl, m, inp, W0, sl, np.arange(T))
        off += T
    assert off == got["seed"].numel()


def test_encode_modules_ragged_groups_with_stale_workspace():
    """Per-element batched encode of modules whose rows end inside a 32-row
    work group, into a workspace whose bytes all start as 0xFF: the re-score
    must read only list entries the screen wrote (every slot, rows past the
    end included) and index the basis tables with seeds below S.  Outputs
    equal those of the same call on a zeroed workspace and of per-module
    calls, and agree with the oracle."""
    wl = workload("block3b", S=24)
    mods = [Module("a", 37, 256, 0, 1, 1), Module("b", 5, 128, 0, 2, 2), Module("c", 70, 384, 0, 3, 3)]
    p = _params(wl)
    inps, W0s = [], []
    for m in mods:
        inp = gen_module_inputs(wl, m, DEV)
        W0s.append(awsrc.awsrc_backbone_rtn(inp["W"])[3])
        inps.append(inp)
    shapes = [(m.rows, m.cols) for m in mods]
    nbytes = awsrc.encode_modules_workspace_bytes(p, shapes, awsrc.AWSRC_DTYPE_BF16, awsrc.AWSRC_D_PER_ELEM)
    outs = []
    for fill in (0xFF, 0x00):
        ws = torch.full((nbytes + 512,), fill, dtype=torch.uint8, device=DEV)
        outs.append(awsrc.awsrc_encode_modules(p, [i["W"] for i in inps], W0s, [i["d"] for i in inps],
                                               want_alpha=True, workspace=ws))
        torch.cuda.synchronize()
    for k in ("seed", "codes", "scale", "gain", "alpha"):
        assert torch.equal(outs[0][k], outs[1][k]), k
    off = 0
    for m, inp, W0 in zip(mods, inps, W0s):
        T = m.rows * m.cols // wl.C
        ref = awsrc.awsrc_encode_tiles(p, inp["W"], W0, inp["d"], want_alpha=True)
        torch.cuda.synchronize()
        for k in ("seed", "codes", "scale", "gain", "alpha"):
            assert torch.equal(outs[0][k][off:off + T], ref[k]), (m.name, k)
        sl = {k: (v[off:off + T] if v is not None and k != "workspace" else v) for k, v in outs[0].items()}
        _check_encode_sample(wl, m, inp, W0, sl, np.arange(T))
        off += T


# ------------------------------------------------------------------ screen error vs the re-score window
@pytest.mark.parametrize("name,rows,cols,S", [("block3b", 256, 2048, 256), ("down3b", 128, 11008, 256),
                                              ("layer32b", 64, 5120, 1024), ("block3b", 11008, 2048, 256)])
def test_screen_error_within_rescore_window(name, rows, cols, S):
    """The fp32 screen's score of the seed the encoder stored against the fp64
    gain of the stored record, over every tile where the screen's best seed
    is the stored one: the difference stays below a tenth of the re-score's
    window (1e-4 |g| + 1e-7 sum d r^2; 3e-2 |g| + 3e-5 sum d r^2 for a
    candidate the screen flagged as a rounding knife edge), so the window
    covers the screen's error tenfold.  (Per-element weights: the batched
    screen; per column at C = 64 with seed ranges, and at C = 128: the
    screens whose lists reach the workspace.)"""
    wl = workload(name, S=S)
    m = Module("win", rows, cols, 0, 1, 1)
    inp, (codes, scale, zero, W0), enc = _gpu_module(wl, m, want_alpha=False)
    d_mode = awsrc.AWSRC_D_PER_COL if inp["d"].dim() == 1 else awsrc.AWSRC_D_PER_ELEM
    g32, w32 = awsrc.awsrc_encode_screen_lists(_params(wl), [(rows, cols)], d_mode, enc["workspace"])
    torch.cuda.synchronize()
    g32 = g32.cpu().numpy().astype(np.float64)
    w32 = w32.cpu().numpy().astype(np.int64)
    # best over the seed ranges: (gain desc, seed asc)
    T, ns, _ = g32.shape
    gg, ss, ff = g32[:, :, 0], w32[:, :, 0] & 0xFFFF, (w32[:, :, 0] >> 16) & 1
    order = np.lexsort((ss, -gg), axis=1)[:, 0]
    gbest, sbest, fbest = gg[np.arange(T), order], ss[np.arange(T), order], ff[np.arange(T), order]
    g64 = enc["gain"].cpu().numpy()
    seed = _u16(enc["seed"])
    r = inp["W32"] - W0
    dd = inp["d"] if inp["d"].dim() == 2 else inp["d"][None, :].expand(rows, cols)
    e = (dd * r * r).reshape(T, wl.C).sum(dim=1).double().cpu().numpy()
    same = seed == sbest
    assert same.mean() > 0.99
    narrow = 1e-4 * np.abs(g64) + 1e-7 * e
    wide = 3e-2 * np.abs(g64) + 3e-5 * e
    diff = np.abs(gbest - g64)
    plain, edge = same & (fbest == 0), same & (fbest == 1)
    rel = diff / np.maximum(np.abs(g64), 1e-30)
    print(f"{name} {rows}x{cols} S={S}: {int(same.sum())} tiles, {int(edge.sum())} flagged; "
          f"largest |g32 - g64| / |g64|: {rel[plain].max():.2e} unflagged "
          f"({(diff / narrow)[plain].max():.3f} of the narrow window), "
          f"{rel[edge].max() if edge.any() else 0.0:.2e} flagged "
          f"({(diff / wide)[edge].max() if edge.any() else 0.0:.3f} of the wide window)")
    assert (diff / narrow)[plain].max() <= 0.1
    if edge.any():
        assert (diff / wide)[edge].max() <= 0.1
