"""Workload recipes and seeded generators.

The paper evaluates on Qwen2.5-3B MLP projections with activation statistics
captured from calibration text and a Fisher diagonal from WikiText-2
gradients (Sec. 4).  None of those are available here, so seeded synthetic
tensors with the same shapes stand in for them:

* weights ~ N(0, std^2), sampled in fp32 and rounded RNE to bf16 where the
  workload stores bf16; optional outlier input channels are multiplied by 8
  after rounding (exact in bf16);
* activation second moments a_j ~ LogNormal(0, sigma), one vector per distinct
  layer input (q/k/v share one, gate/up share one, o and down own one);
* a diagonal Fisher proxy F_ij = mean of 64 squared N(0,1) gradients, drawn
  directly from its exact law Gamma(shape=32, rate=32);
* per-element blended weights d_ij = 0.5 a_j + 0.5 F_ij (the Fisher/activation
  blend of the P_F variant, Sec. 3.3), or per-column d_j = a_j.

Every tensor is drawn from its own generator seeded with
``layer*1000 + module_index*10 + field`` (field 0 = W, 1 = outlier set,
2 = a, 3 = Fisher), so a module's inputs do not depend on which other
modules were generated first.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional, Tuple

import torch

FIELD_W, FIELD_OUTLIER, FIELD_ACT, FIELD_FISHER = 0, 1, 2, 3


@dataclasses.dataclass(frozen=True)
class Module:
    name: str
    rows: int          # output features (rows of W)
    cols: int          # input features (tiles run along this dimension)
    layer: int         # decoder layer index (seed base)
    index: int         # module index within its layer
    act_index: int     # module index whose seed draws this module's activation vector


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    description: str
    modules: Tuple[Module, ...]
    w_dtype: str               # "f32" | "bf16"
    w_std: float
    outlier_frac: float
    a_sigma: float
    d_mode: str                # "col" (activation only) | "elem" (Fisher blend)
    C: int
    P: int
    b: int
    S: int
    mode: str                  # "global" (P variant) | "per_module" (U variant)
    budgets: Tuple[float, ...]  # bits/weight budgets decoded from one ranked stream
    basis_key: int = 0
    ridge_lambda: float = 1e-6
    idx_bits: int = 32

    @property
    def n_weights(self) -> int:
        return sum(m.rows * m.cols for m in self.modules)

    @property
    def n_tiles(self) -> int:
        return sum(m.rows * m.cols // self.C for m in self.modules)

    @property
    def candidates(self) -> int:
        return self.n_tiles * self.S


def round_half_even_count(frac: float, n: int) -> int:
    """Number of outlier channels: frac*n rounded half-to-even."""
    return int(round(frac * n))


def _block_modules(layer: int, hidden: int, kv: int, inter: int) -> Tuple[Module, ...]:
    # q, k, v share the attention input; gate, up share the MLP input.
    spec = [("q_proj", hidden, hidden, 0), ("k_proj", kv, hidden, 0),
            ("v_proj", kv, hidden, 0), ("o_proj", hidden, hidden, 3),
            ("gate_proj", inter, hidden, 4), ("up_proj", inter, hidden, 4),
            ("down_proj", hidden, inter, 6)]
    return tuple(Module(f"layers.{layer}.{n}", r, c, layer, i, a)
                 for i, (n, r, c, a) in enumerate(spec))


def _make_workloads() -> Dict[str, Workload]:
    w = {}
    w["linear256"] = Workload(
        name="linear256",
        description="single fp32 256x256 linear layer, C=64 S=64 P=4 b=4, global prefix at 0.162 bpw",
        modules=(Module("linear", 256, 256, 0, 0, 0),),
        w_dtype="f32", w_std=0.02, outlier_frac=0.0, a_sigma=1.0, d_mode="col",
        C=64, P=4, b=4, S=64, mode="global", budgets=(0.162,))
    w["down3b"] = Workload(
        name="down3b",
        description="3B-model MLP down projection 2048x11008 bf16 with 1% x8 outlier channels, "
                    "C=64 S=256 P=8 b=4, per-module quota of 0.162 bpw",
        modules=(Module("mlp.down_proj", 2048, 11008, 0, 0, 0),),
        w_dtype="bf16", w_std=0.02, outlier_frac=0.01, a_sigma=1.5, d_mode="col",
        C=64, P=8, b=4, S=256, mode="per_module", budgets=(0.162,))
    w["block3b"] = Workload(
        name="block3b",
        description="3B-model decoder block (q,k,v,o,gate,up,down), bf16, Fisher/activation blend, "
                    "C=64 S=256 P=8 b=4, global prefixes at 0.08/0.162/0.32 bpw",
        modules=_block_modules(0, 2048, 256, 11008),
        w_dtype="bf16", w_std=0.02, outlier_frac=0.0, a_sigma=1.5, d_mode="elem",
        C=64, P=8, b=4, S=256, mode="global", budgets=(0.08, 0.162, 0.32))
    w["layer32b"] = Workload(
        name="layer32b",
        description="32B-model decoder layer, bf16 with 0.5% x8 outlier channels, "
                    "C=128 S=1024 P=8 b=3, global prefix at 0.162 bpw",
        modules=_block_modules(0, 5120, 1024, 27648),
        w_dtype="bf16", w_std=0.015, outlier_frac=0.005, a_sigma=2.0, d_mode="col",
        C=128, P=8, b=3, S=1024, mode="global", budgets=(0.162,))
    w["stack3b"] = Workload(
        name="stack3b",
        description="36-layer 3B-model stack of block3b layers (layer seeds 0..35), "
                    "C=64 S=512 P=8 b=4, one global ranking, prefixes at 0.04/0.08/0.162/0.32 bpw",
        modules=tuple(m for L in range(36) for m in _block_modules(L, 2048, 256, 11008)),
        w_dtype="bf16", w_std=0.02, outlier_frac=0.0, a_sigma=1.5, d_mode="elem",
        C=64, P=8, b=4, S=512, mode="global", budgets=(0.04, 0.08, 0.162, 0.32))
    return w


WORKLOADS: Dict[str, Workload] = _make_workloads()


def workload(name: str, **overrides) -> Workload:
    """Look up a workload; keyword overrides give scaled-down variants for tests."""
    wl = WORKLOADS[name]
    return dataclasses.replace(wl, **overrides) if overrides else wl


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def _seed(m: Module, field: int, index: Optional[int] = None) -> int:
    return m.layer * 1000 + (m.index if index is None else index) * 10 + field


def gen_weight(wl: Workload, m: Module, device="cpu") -> torch.Tensor:
    """W [rows, cols] in the workload's storage dtype (fp32 or bf16)."""
    g = _gen(_seed(m, FIELD_W), device)
    w = torch.randn(m.rows, m.cols, generator=g, device=device, dtype=torch.float32)
    w.mul_(wl.w_std)
    if wl.w_dtype == "bf16":
        w = w.to(torch.bfloat16)
    n_out = round_half_even_count(wl.outlier_frac, m.cols)
    if n_out:
        go = _gen(_seed(m, FIELD_OUTLIER), device)
        cols = torch.randperm(m.cols, generator=go, device=device)[:n_out]
        w[:, cols] = w[:, cols] * 8
    return w


def gen_activation(wl: Workload, m: Module, device="cpu") -> torch.Tensor:
    """a_j = E[x_j^2] stand-in: LogNormal(0, a_sigma) over the module's input channels."""
    g = _gen(_seed(m, FIELD_ACT, m.act_index), device)
    z = torch.randn(m.cols, generator=g, device=device, dtype=torch.float32)
    return torch.exp(z * wl.a_sigma)


def gen_fisher(wl: Workload, m: Module, device="cpu") -> torch.Tensor:
    """Per-element Fisher proxy: mean of 64 squared N(0,1) draws ~ Gamma(32, rate 32)."""
    seed = _seed(m, FIELD_FISHER)
    dv = torch.device(device)
    devs = [dv.index if dv.index is not None else torch.cuda.current_device()] if dv.type == "cuda" else []
    with torch.random.fork_rng(devices=devs):
        torch.manual_seed(seed)
        if devs:
            torch.cuda.manual_seed(seed)
        conc = torch.full((m.rows, m.cols), 32.0, device=device, dtype=torch.float32)
        f = torch._standard_gamma(conc)
    return f / 32.0


def gen_module_inputs(wl: Workload, m: Module, device="cpu") -> Dict[str, torch.Tensor]:
    """Inputs of one module: W (storage dtype), W32 (same values in fp32) and d.

    d is [cols] (per input channel, shared across rows) for d_mode "col" and
    [rows, cols] for the per-element Fisher blend.
    """
    W = gen_weight(wl, m, device)
    a = gen_activation(wl, m, device)
    if wl.d_mode == "col":
        d = a.contiguous()
    else:
        F = gen_fisher(wl, m, device)
        d = (0.5 * a)[None, :] + 0.5 * F
    return {"W": W, "W32": W.to(torch.float32), "d": d.contiguous()}


def gen_records(T: int, P: int, b: int, S: int, seed: int, device="cpu",
                frac_nonpositive: float = 0.3, frac_ties: float = 0.1) -> Dict[str, torch.Tensor]:
    """Random per-tile records shaped like encoder outputs, for ranking and
    decoding tests: seeds in [0, S), codes in [-qmax, qmax], positive finite
    fp16 scale bit patterns, fp64 gains with a share of non-positive values
    and a share of exactly repeated values (ties)."""
    g = _gen(seed, device)
    qmax = (1 << (b - 1)) - 1
    seeds = torch.randint(0, S, (T,), generator=g, device=device, dtype=torch.int64)
    codes = torch.randint(-qmax, qmax + 1, (T, P), generator=g, device=device, dtype=torch.int64)
    scale = torch.randint(0x0400, 0x2C00, (T,), generator=g, device=device, dtype=torch.int64)
    gain = torch.exp(torch.randn(T, generator=g, device=device, dtype=torch.float64) * 2.0 - 12.0)
    u = torch.rand(T, generator=g, device=device, dtype=torch.float64)
    gain = torch.where(u < frac_nonpositive * 0.5, -gain, gain)
    gain = torch.where((u >= frac_nonpositive * 0.5) & (u < frac_nonpositive), torch.zeros_like(gain), gain)
    v = torch.rand(T, generator=g, device=device, dtype=torch.float64)
    tie_val = torch.exp(torch.randint(-14, -10, (T,), generator=g, device=device).to(torch.float64))
    gain = torch.where((v < frac_ties) & (u >= frac_nonpositive), tie_val, gain)
    return {"seed": seeds.to(torch.int16), "codes": codes.to(torch.int8), "scale": scale.to(torch.int16),
            "gain": gain}
