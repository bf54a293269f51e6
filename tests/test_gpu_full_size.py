"""Parity of the HIP path with the oracle at the workloads' full sizes.

* 3B down projection (2048 x 11008, per-column weights, S = 256): every one
  of its 352,256 tiles against the oracle.
* 3B decoder block (seven modules, per-element weights, S = 256): every tile
  of every module, and the global-ranking chain of Sec. 3.3: one ranking of
  the encoder's own records, the 0.08 and 0.162 bits/weight streams byte
  prefixes of the 0.32 one and equal to the oracle's streams built from the
  same records, every prefix decoded against the oracle's decoder.
* 32B decoder layer (seven modules, C = 128, S = 1024) and the 36-layer 3B
  stack (252 modules, S = 512): every 256th row of every module (all of that
  row's tiles) against the oracle; for the stack also one global ranking of
  all 43.35M tiles' records at 0.32 bits/weight, the 0.04/0.08/0.162 streams
  as its byte prefixes, and every prefix decoded (dense bf16 reconstruction,
  and in place onto fp32 W0 for the largest) on the sampled rows.

The oracle runs over worker processes (tests/oracle_pool.py); the bars are
those of the encoder parity tests.  Inputs are the seeded workload
generators' tensors; the oracle computes its own backbone and residual.
"""
import numpy as np
import pytest
import torch

import oracle_pool as OP
from oracle import awsrc_oracle as O
from synth import WORKLOADS, gen_module_inputs

pytestmark = pytest.mark.gpu

awsrc = pytest.importorskip("paper_2608_23144_amd")

DEV = "cuda"
ROW_STEP = 256  # row sample of the two largest workloads


def _u16(t):
    return (t.to(torch.int32) & 0xFFFF).cpu().numpy()


def _params(wl):
    return awsrc.make_params(wl.C, wl.P, wl.b, wl.S, basis_key=wl.basis_key, ridge_lambda=wl.ridge_lambda,
                             idx_bits=wl.idx_bits)


def _oparams(wl):
    return O.Params(C=wl.C, P=wl.P, b=wl.b, S=wl.S, basis_key=wl.basis_key, ridge_lambda=wl.ridge_lambda,
                    idx_bits=wl.idx_bits)


class Encoded:
    """GPU backbone and encoder outputs of every module of a workload, the
    outputs concatenated in module order (global tile order)."""

    def __init__(self, wl, rows_of=None, keep_W0=False, keep_backbone=False, want_alpha=True):
        self.wl = wl
        self.shapes = [(m.rows, m.cols) for m in wl.modules]
        T = wl.n_tiles
        self.seed = torch.empty(T, dtype=torch.int16, device=DEV)
        self.codes = torch.empty(T, wl.P, dtype=torch.int8, device=DEV)
        self.scale = torch.empty(T, dtype=torch.int16, device=DEV)
        self.gain = torch.empty(T, dtype=torch.float64, device=DEV)
        self.alpha = torch.empty(T, wl.P, dtype=torch.float32, device=DEV) if want_alpha else None
        self.toff = np.cumsum([0] + [r * c // wl.C for r, c in self.shapes])
        self.W0, self.bb, self.host = [], [], []
        p = _params(wl)
        for i, m in enumerate(wl.modules):
            inp = gen_module_inputs(wl, m, DEV)
            codes, scale, zero, W0 = awsrc.awsrc_backbone_rtn(inp["W"])
            sl = slice(int(self.toff[i]), int(self.toff[i + 1]))
            out = {"seed": self.seed[sl], "codes": self.codes[sl], "scale": self.scale[sl], "gain": self.gain[sl],
                   "alpha": None if self.alpha is None else self.alpha[sl]}
            awsrc.awsrc_encode_tiles(p, inp["W"], W0, inp["d"], out=out)
            rows = np.arange(m.rows) if rows_of is None else rows_of(m)
            ri = torch.as_tensor(rows, device=DEV)
            # host copies of the sampled rows' inputs (fp32 W, d) and the GPU's W0 there
            self.host.append({"rows": rows, "W32": inp["W32"][ri].cpu().numpy(),
                              "d": (inp["d"] if inp["d"].dim() == 1 else inp["d"][ri]).cpu().numpy(),
                              "W0_gpu": W0[ri].cpu().numpy()})
            if keep_W0:
                self.W0.append(W0)
            if keep_backbone:
                self.bb.append((codes, scale, zero))
            del inp
        torch.cuda.synchronize()

    def sample_tiles(self, i):
        """Global tile indices of module i's sampled rows, row-major."""
        m = self.wl.modules[i]
        nb = m.cols // self.wl.C
        rows = self.host[i]["rows"]
        return (self.toff[i] + rows[:, None] * nb + np.arange(nb)[None, :]).ravel()

    def jobs(self, i, n_chunks):
        """Oracle comparison jobs for module i's sampled rows (the oracle's own
        backbone of those rows, checked bit-exact against the GPU's W0)."""
        wl, m, hs = self.wl, self.wl.modules[i], self.host[i]
        _, _, _, W0o = O.rtn_backbone(hs["W32"])
        assert np.array_equal(W0o, hs["W0_gpu"]), f"backbone of {m.name}"
        R = O.tiles(O.residual(hs["W32"], W0o), wl.C)
        D = O.tile_weights(hs["d"], len(hs["rows"]), m.cols, wl.C)
        t = torch.as_tensor(self.sample_tiles(i), device=DEV)
        return OP.chunk_jobs(m.name, R, D, _oparams(wl), _u16(self.seed[t]), self.codes[t].cpu().numpy(),
                             _u16(self.scale[t]), self.gain[t].cpu().numpy(),
                             None if self.alpha is None else self.alpha[t].cpu().numpy(), n_chunks)

    def rank(self, bpw):
        return awsrc.awsrc_rank_prefix(_params(self.wl), self.shapes, awsrc.AWSRC_MODE_GLOBAL, bpw, self.seed,
                                       self.codes, self.scale, self.gain)

    def records(self):
        return {"seed": _u16(self.seed).astype(np.int64), "codes": self.codes.cpu().numpy().astype(np.int64),
                "scale": _u16(self.scale).astype(np.int64), "gain": self.gain.cpu().numpy()}


def _assert_parity(tot, what):
    msg = (f"{what}: {tot['tiles']} tiles, {tot['seed_diff']} tied seeds, {tot['edge']} knife-edge records, "
           f"{tot['failures']} failures; oracle {tot['cpu_seconds']:.0f} CPU-s over {tot['workers']} workers")
    print(msg)
    assert tot["failures"] == 0, msg + "\n" + "\n".join(tot["report"])
    # exact ties are rare; many tied seeds would point at a screen that
    # systematically misses the best seed by less than the window
    assert tot["seed_diff"] <= max(2, tot["tiles"] // 200), msg


def _every_nth_row(n):
    return lambda m: np.arange(0, m.rows, n)


# ------------------------------------------------------------ 3B down projection
def test_down3b_every_tile():
    wl = WORKLOADS["down3b"]
    enc = Encoded(wl)
    tot = OP.run_jobs(enc.jobs(0, 4 * OP.n_workers()))
    assert tot["tiles"] == wl.n_tiles
    _assert_parity(tot, "down3b")


# ------------------------------------------------------------ 3B decoder block
@pytest.fixture(scope="module")
def block3b():
    enc = Encoded(WORKLOADS["block3b"], keep_W0=True)
    yield enc
    del enc
    torch.cuda.empty_cache()


@pytest.mark.parametrize("mi", range(7))
def test_block3b_every_tile(block3b, mi):
    m = block3b.wl.modules[mi]
    n = max(1, min(4 * OP.n_workers(), m.rows * m.cols // block3b.wl.C // 2048))
    tot = OP.run_jobs(block3b.jobs(mi, n))
    assert tot["tiles"] == m.rows * m.cols // block3b.wl.C
    _assert_parity(tot, m.name)


def test_block3b_nested_prefixes_match_oracle(block3b):
    """One global ranking at 0.32 bits/weight; the 0.08 and 0.162 streams are
    its byte prefixes and equal the oracle's streams of the same records;
    each decodes (in place, fp32 W0) as the oracle's decoder does."""
    enc = block3b
    wl = enc.wl
    op = _oparams(wl)
    rec = enc.records()
    streams = {}
    for bpw in (0.32, 0.162, 0.08):
        s, K, ne = enc.rank(bpw)
        want, K_o, ne_o = O.build_stream(op, enc.shapes, rec, bpw, per_module=False)
        assert (K, ne) == (K_o, ne_o), bpw
        got = bytes(s.cpu().numpy().tobytes())
        assert got == want, bpw
        streams[bpw] = (s, got, K)
    full = streams[0.32][1]
    for bpw in (0.162, 0.08):
        assert full[:len(streams[bpw][1])] == streams[bpw][1], bpw
        assert streams[bpw][2] < streams[0.32][2]
    W0s = [w.cpu().numpy() for w in enc.W0]
    for bpw in (0.08, 0.162, 0.32):
        s, stream, K = streams[bpw]
        ref = O.decode_add(stream, W0s)
        dev = [w.clone() for w in enc.W0]
        awsrc.awsrc_decode_add(s, dev)
        for w0, got, want in zip(W0s, dev, ref):
            got = got.cpu().numpy()
            w0f = w0.astype(np.float64)
            mag = np.abs(w0f) + np.abs(want - w0f)
            assert np.all(np.abs(got - want) <= 2.0 ** -22 * mag + 1e-30), bpw
            moved = got != w0
            assert moved.sum() <= K * wl.C
        del dev


# ------------------------------------------------------------ 32B decoder layer
def test_layer32b_row_sample():
    wl = WORKLOADS["layer32b"]
    enc = Encoded(wl, rows_of=_every_nth_row(ROW_STEP))
    jobs = [j for i in range(len(wl.modules)) for j in enc.jobs(i, 8)]
    tot = OP.run_jobs(jobs)
    assert tot["tiles"] == sum(len(range(0, m.rows, ROW_STEP)) * (m.cols // wl.C) for m in wl.modules)
    _assert_parity(tot, "layer32b, every 256th row")
    del enc
    torch.cuda.empty_cache()


# ------------------------------------------------------------ 36-layer 3B stack
@pytest.fixture(scope="module")
def stack3b():
    enc = Encoded(WORKLOADS["stack3b"], rows_of=_every_nth_row(ROW_STEP), keep_W0=True, keep_backbone=True,
                  want_alpha=False)
    yield enc
    del enc
    torch.cuda.empty_cache()


def test_stack3b_row_sample(stack3b):
    wl = stack3b.wl
    jobs = [j for i in range(len(wl.modules)) for j in stack3b.jobs(i, 1)]
    tot = OP.run_jobs(jobs)
    assert tot["tiles"] == sum(len(range(0, m.rows, ROW_STEP)) * (m.cols // wl.C) for m in wl.modules)
    _assert_parity(tot, "stack3b, every 256th row")


def _sampled_records(enc, stream, K, hd):
    """Records of a stream whose tiles lie on the sampled rows: (module,
    row position in the sample, column block, seed, codes, scale field)."""
    L, h = hd["L_rec"], hd["h"]
    raw = np.frombuffer(stream, dtype=np.uint8, offset=h, count=K * L).reshape(K, L)
    assert hd["idx_bits"] == 32
    tiles = raw[:, :4].copy().view("<u4").ravel().astype(np.int64)
    mi = np.searchsorted(enc.toff, tiles, side="right") - 1
    nb = np.array([m.cols // enc.wl.C for m in enc.wl.modules], dtype=np.int64)[mi]
    row, blk = np.divmod(tiles - enc.toff[mi], nb)
    out = []
    for k in np.flatnonzero(row % ROW_STEP == 0):
        t, s, codes, sc = O.unpack_record(bytes(raw[k]), hd["idx_bits"], hd["seed_bits"], hd["P"], hd["b"],
                                          hd["scale_bits"])
        assert t == tiles[k]
        out.append((int(mi[k]), int(row[k]) // ROW_STEP, int(blk[k]), s, np.asarray(codes, dtype=np.float64), sc))
    return out


def _oracle_rows(enc, recs, hd):
    """The oracle's repaired sampled rows: its own backbone W0 of those rows
    plus B_s (scale q) for every record on them, in fp64 (Eq. (1), Sec. 3.2)."""
    C, P = enc.wl.C, enc.wl.P
    W0o = [O.rtn_backbone(hs["W32"])[3] for hs in enc.host]
    out = [w.astype(np.float64) for w in W0o]
    touched = [np.zeros((w.shape[0], w.shape[1] // C), bool) for w in W0o]
    cache = {}
    for mi, r, blk, s, codes, sc in recs:
        if s not in cache:
            cache[s] = O.basis_matrix(hd["basis_key"], s, C, P, hd["gen_version"])
        scv = float(np.array([sc], dtype=np.uint16).view(np.float16)[0])
        out[mi][r, blk * C:(blk + 1) * C] += cache[s] @ (scv * codes)
        touched[mi][r, blk] = True
    return W0o, out, touched


def test_stack3b_nested_prefixes(stack3b):
    """One global ranking of every tile of the 36-layer stack at 0.32
    bits/weight (Sec. 4: a single ranking, prefixes at each rate); the
    0.04/0.08/0.162 streams are its byte prefixes with K from each budget; the
    record order equals an independent numpy ordering by (-gain, tile); every
    prefix is decoded without re-encoding, densely to bf16 from the stored
    backbone, and the largest also in place onto fp32 W0, and the sampled rows
    agree with the oracle."""
    enc = stack3b
    wl = enc.wl
    op = _oparams(wl)
    T = wl.n_tiles
    N = wl.n_weights
    L = O.record_bytes(op, T)
    h = O.header_bytes(len(enc.shapes))
    streams = {}
    for bpw in (0.32, 0.162, 0.08, 0.04):
        s, K, ne = enc.rank(bpw)
        assert K == min(ne, (O.budget_bytes(bpw, N) - h) // L), bpw
        assert s.numel() == h + K * L
        streams[bpw] = (s, K)
    s32, K32 = streams[0.32]
    for bpw in (0.162, 0.08, 0.04):
        s, K = streams[bpw]
        assert K < K32 and torch.equal(s32[:s.numel()], s), bpw
    # record order: the top K32 eligible tiles by (-gain, tile)
    gain = enc.gain.cpu().numpy()
    elig = np.nonzero(gain > 0)[0]
    g = gain[elig]
    v = -np.partition(-g, K32 - 1)[K32 - 1]
    above = elig[g > v]
    eq = elig[g == v]
    chosen = np.concatenate([above, eq[:K32 - len(above)]])
    want = chosen[np.lexsort((chosen, -gain[chosen]))]
    full = bytes(s32.cpu().numpy().tobytes())
    got = np.frombuffer(full, dtype=np.uint8, offset=h).reshape(K32, L)[:, :4].copy().view("<u4").ravel()
    assert np.array_equal(got.astype(np.int64), want)
    hd = O.parse_header(full[:h])
    # every prefix, reconstructed densely in bf16 (one bf16 buffer set reused)
    outs = [torch.empty(r, c, dtype=torch.bfloat16, device=DEV) for r, c in enc.shapes]
    rows_t = [torch.as_tensor(hs["rows"], device=DEV) for hs in enc.host]
    for bpw in (0.04, 0.08, 0.162, 0.32):
        s, K = streams[bpw]
        plan, ws = awsrc.awsrc_decode_prepare(s, outs)
        awsrc.awsrc_reconstruct_bf16(plan, enc.bb, 128)
        recs = _sampled_records(enc, full, K, hd)
        W0o, ref, touched = _oracle_rows(enc, recs, hd)
        n_rec = n_exact = 0
        for o, ri, w0, rf, tm in zip(outs, rows_t, W0o, ref, touched):
            got = o[ri].to(torch.float32).cpu().numpy().astype(np.float64)
            want_b = O.bf16_round(rf)
            mask = np.repeat(tm, wl.C, axis=1)
            assert np.array_equal(got[~mask], want_b[~mask]), bpw
            # bars of the dense reconstruction tests: one bf16 ulp, the fp32
            # add, and the oracle's own fp64 residue where the exact sum is 0
            w0f = w0.astype(np.float64)
            rh = np.abs(rf - w0f)
            tile_max = np.repeat(rh.reshape(rh.shape[0], -1, wl.C).max(axis=2), wl.C, axis=1)
            mag = np.abs(w0f) + rh
            diff = np.abs(got - want_b)
            assert np.all(diff[mask] <= 2.0 ** -7 * np.abs(want_b[mask]) + 2.0 ** -21 * mag[mask]
                          + 2.0 ** -40 * tile_max[mask]), bpw
            n_rec += int(mask.sum())
            n_exact += int((diff[mask] == 0).sum())
        assert n_rec == len(recs) * wl.C and len(recs) > 0
        assert n_exact >= 0.98 * n_rec
        del plan, ws
    del outs
    torch.cuda.empty_cache()
    # the largest prefix in place onto the fp32 backbone
    awsrc.awsrc_decode_add(s32, enc.W0)
    recs = _sampled_records(enc, full, K32, hd)
    W0o, ref, touched = _oracle_rows(enc, recs, hd)
    for w, ri, w0, rf, tm in zip(enc.W0, rows_t, W0o, ref, touched):
        got = w[ri].cpu().numpy()
        mask = np.repeat(tm, wl.C, axis=1)
        assert np.array_equal(got[~mask], w0[~mask])
        w0f = w0.astype(np.float64)
        assert np.all(np.abs(got - rf)[mask] <= 2.0 ** -22 * (np.abs(w0f) + np.abs(rf - w0f))[mask] + 1e-30)
