"""The allocation-free encoder entry point (awsrc_encode_tiles_noalloc)
against awsrc_encode_tiles with a workspace: identical outputs on two calls
in a row, the second on a smaller module, through the C ABI; a module whose
scratch need exceeds the fixed array is refused."""
import pytest
import torch

from synth import WORKLOADS, Module, gen_module_inputs, workload

pytestmark = pytest.mark.gpu

awsrc = pytest.importorskip("paper_2608_23144_amd")

DEV = "cuda"


def _params(wl, **kw):
    return awsrc.make_params(wl.C, wl.P, wl.b, wl.S, basis_key=wl.basis_key, ridge_lambda=wl.ridge_lambda,
                             idx_bits=wl.idx_bits, **kw)


def _outs(T, P, fill):
    return {"seed": torch.full((T,), fill, dtype=torch.int16, device=DEV),
            "codes": torch.full((T, P), fill, dtype=torch.int8, device=DEV),
            "scale": torch.full((T,), fill, dtype=torch.int16, device=DEV),
            "gain": torch.full((T,), float("nan"), dtype=torch.float64, device=DEV),
            "alpha": torch.full((T, P), float("nan"), dtype=torch.float32, device=DEV)}


def _same(a, b):
    for k in ("seed", "codes", "scale", "alpha"):
        assert torch.equal(a[k], b[k]), k
    assert torch.equal(a["gain"].view(torch.int64), b["gain"].view(torch.int64))


def test_noalloc_encode_matches_workspace_entry_point():
    cases = [
        (WORKLOADS["down3b"], WORKLOADS["down3b"].modules[0]),          # 352,256 tiles, per-column weights
        (workload("block3b", S=40), Module("small", 67, 512, 0, 1, 1)),  # 536 tiles, per-element weights
    ]
    for wl, m in cases:
        inp = gen_module_inputs(wl, m, DEV)
        _, _, _, W0 = awsrc.awsrc_backbone_rtn(inp["W"])
        p = _params(wl)
        T = m.rows * m.cols // wl.C
        ref = awsrc.awsrc_encode_tiles(p, inp["W"], W0, inp["d"], out=_outs(T, wl.P, -1))
        got = awsrc.awsrc_encode_tiles_noalloc(p, inp["W"], W0, inp["d"], out=_outs(T, wl.P, 0x55))
        torch.cuda.synchronize()
        _same(ref, got)


def test_noalloc_encode_refuses_oversized_scratch():
    wl = workload("down3b", S=65536)
    m = WORKLOADS["down3b"].modules[0]
    W = torch.empty(m.rows, m.cols, dtype=torch.bfloat16, device=DEV)
    W0 = torch.empty(m.rows, m.cols, dtype=torch.float32, device=DEV)
    d = torch.ones(m.cols, dtype=torch.float32, device=DEV)
    T = m.rows * m.cols // wl.C
    with pytest.raises(awsrc.AwsrcError) as ei:
        awsrc.awsrc_encode_tiles_noalloc(_params(wl), W, W0, d, out=_outs(T, wl.P, 0))
    assert ei.value.status == awsrc.AWSRC_ENOSPC
