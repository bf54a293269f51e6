"""Python binding of libawsrc, the HIP (gfx950) implementation of the AWSRC
encoder/decoder hot path.

The functions carry the names of the C entry points declared in
include/awsrc.h and only marshal arguments: torch allocates the device
buffers and supplies the stream; every step of the codec runs in the
library's kernels.  Importing this module fails loudly if the library has
not been built (python paper_2608_23144_amd/build.py).
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libawsrc.so")

AWSRC_OK, AWSRC_EINVAL, AWSRC_ENOSPC, AWSRC_ECORRUPT, AWSRC_EDEVICE = 0, -1, -2, -3, -4
AWSRC_DTYPE_F32, AWSRC_DTYPE_BF16 = 0, 1
AWSRC_D_PER_COL, AWSRC_D_PER_ELEM = 0, 1
AWSRC_MODE_GLOBAL, AWSRC_MODE_PER_MODULE = 0, 1
AWSRC_SCALE_FP16, AWSRC_SCALE_POW2 = 0, 1

EXPORTED = ("awsrc_abi_version", "awsrc_last_error", "awsrc_backbone_rtn", "awsrc_sdq_encode",
            "awsrc_backbone_sdq_dequant", "awsrc_encode_tiles",
            "awsrc_encode_modules", "awsrc_encode_screen_lists", "awsrc_encode_tiles_noalloc", "awsrc_encode_noalloc_max_bytes",
            "awsrc_encode_scored", "awsrc_rank_prefix", "awsrc_decode_add", "awsrc_decode_prepare", "awsrc_decode_apply",
            "awsrc_reconstruct_bf16", "awsrc_reconstruct_bf16_prefixes", "awsrc_reconstruct_bf16_sdq", "awsrc_record_bytes", "awsrc_header_bytes", "awsrc_budget_bytes", "awsrc_prefix_K")


class AwsrcError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"awsrc status {status}: {msg}")
        self.status = status


class awsrc_params(ctypes.Structure):
    _fields_ = [("C", ctypes.c_int32), ("P", ctypes.c_int32), ("b", ctypes.c_int32), ("S", ctypes.c_int32),
                ("scale_fmt", ctypes.c_int32), ("idx_bits", ctypes.c_int32), ("gen_version", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("basis_key", ctypes.c_uint64), ("ridge_lambda", ctypes.c_double)]


class awsrc_decode_plan(ctypes.Structure):
    _fields_ = [("C", ctypes.c_int32), ("P", ctypes.c_int32), ("b", ctypes.c_int32), ("S", ctypes.c_int32),
                ("idx_bits", ctypes.c_int32), ("seed_bits", ctypes.c_int32), ("L_rec", ctypes.c_int32),
                ("n_modules", ctypes.c_int32), ("w0_dtype", ctypes.c_int32), ("scale_fmt", ctypes.c_int32),
                ("K", ctypes.c_int64), ("T_total", ctypes.c_uint64), ("h", ctypes.c_uint64),
                ("records", ctypes.c_void_p), ("workspace", ctypes.c_void_p)]


def make_params(C: int, P: int, b: int, S: int, basis_key: int = 0, ridge_lambda: float = 1e-6,
                idx_bits: int = 32, scale_fmt: int = AWSRC_SCALE_FP16, gen_version: int = 1) -> awsrc_params:
    return awsrc_params(C, P, b, S, scale_fmt, idx_bits, gen_version, 0, basis_key, ridge_lambda)


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python paper_2608_23144_amd/build.py`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, u64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_size_t
    pp = ctypes.POINTER(awsrc_params)
    P64 = ctypes.POINTER(ctypes.c_int64)
    sig = {
        "awsrc_abi_version": (i32, []),
        "awsrc_last_error": (ctypes.c_char_p, []),
        "awsrc_backbone_rtn": (i32, [vp, i32, i64, i64, i32, vp, vp, vp, vp, vp]),
        "awsrc_sdq_encode": (i32, [vp, i64, vp, vp, vp, vp]),
        "awsrc_backbone_sdq_dequant": (i32, [vp, vp, vp, vp, vp, i64, i64, i32, vp, vp]),
        "awsrc_encode_tiles": (i32, [pp, vp, i32, vp, i64, i64, vp, i32, vp, vp, vp, vp, vp, vp,
                                     ctypes.POINTER(sz), vp]),
        "awsrc_encode_modules": (i32, [pp, i32, ctypes.POINTER(vp), i32, ctypes.POINTER(vp), ctypes.POINTER(vp), i32,
                                       P64, P64, vp, vp, vp, vp, vp, vp, ctypes.POINTER(sz), vp]),
        "awsrc_encode_screen_lists": (i32, [pp, i32, P64, P64, i32, vp, vp, vp, ctypes.POINTER(i32), vp]),
        "awsrc_encode_tiles_noalloc": (i32, [pp, vp, i32, vp, i64, i64, vp, i32, vp, vp, vp, vp, vp, vp]),
        "awsrc_encode_noalloc_max_bytes": (u64, []),
        "awsrc_encode_scored": (i32, [vp, ctypes.POINTER(u64), vp]),
        "awsrc_rank_prefix": (i32, [pp, i32, P64, P64, i32, ctypes.c_double, vp, vp, vp, vp, vp, u64,
                                    ctypes.POINTER(u64), P64, P64, vp, ctypes.POINTER(sz), vp]),
        "awsrc_decode_add": (i32, [vp, u64, i32, ctypes.POINTER(vp), P64, P64, i32, vp,
                                   ctypes.POINTER(sz), vp]),
        "awsrc_decode_prepare": (i32, [vp, u64, i32, ctypes.POINTER(vp), P64, P64, i32,
                                       ctypes.POINTER(awsrc_decode_plan), vp, ctypes.POINTER(sz), vp]),
        "awsrc_decode_apply": (i32, [ctypes.POINTER(awsrc_decode_plan), vp]),
        "awsrc_reconstruct_bf16": (i32, [ctypes.POINTER(awsrc_decode_plan), i32, ctypes.POINTER(vp),
                                         ctypes.POINTER(vp), ctypes.POINTER(vp), vp]),
        "awsrc_reconstruct_bf16_prefixes": (i32, [ctypes.POINTER(awsrc_decode_plan), i32, P64, ctypes.POINTER(vp),
                                                  i32, ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp),
                                                  vp]),
        "awsrc_reconstruct_bf16_sdq": (i32, [ctypes.POINTER(awsrc_decode_plan), i32, P64, ctypes.POINTER(vp), i32,
                                             ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp),
                                             ctypes.POINTER(vp), ctypes.POINTER(vp), vp]),
        "awsrc_record_bytes": (i64, [pp, i64]),
        "awsrc_header_bytes": (i64, [i32]),
        "awsrc_budget_bytes": (i64, [ctypes.c_double, i64]),
        "awsrc_prefix_K": (i64, [i64, i64, i64, i64]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype, f.argtypes = res, args
    return lib


LIB = _load()


def _check(status: int) -> None:
    if status != AWSRC_OK:
        raise AwsrcError(status, LIB.awsrc_last_error().decode(errors="replace"))


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return AWSRC_DTYPE_F32
    if t.dtype == torch.bfloat16:
        return AWSRC_DTYPE_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _dev(*ts):
    for t in ts:
        if t is not None and (not t.is_cuda or not t.is_contiguous()):
            raise ValueError("tensors must be contiguous device tensors")


def _workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


# ------------------------------------------------------------------ host-only helpers
def awsrc_abi_version() -> int:
    return LIB.awsrc_abi_version()


def awsrc_record_bytes(p: awsrc_params, T_total: int) -> int:
    return LIB.awsrc_record_bytes(ctypes.byref(p), T_total)


def awsrc_header_bytes(n_modules: int) -> int:
    return LIB.awsrc_header_bytes(n_modules)


def awsrc_budget_bytes(bpw: float, n_weights: int) -> int:
    return LIB.awsrc_budget_bytes(bpw, n_weights)


def awsrc_prefix_K(budget_bytes: int, h: int, L_rec: int, n_eligible: int) -> int:
    return LIB.awsrc_prefix_K(budget_bytes, h, L_rec, n_eligible)


# ------------------------------------------------------------------ device calls
def awsrc_backbone_rtn(W: torch.Tensor, group: int = 128, want_W0: bool = True, out=None, stream=None):
    """RTN-INT4 backbone; returns (codes u8, scale fp16-bits i16-view, zero u8, W0 fp32 or None)."""
    _dev(W)
    rows, cols = W.shape
    if out is None:
        dev = W.device
        out = (torch.empty(rows, cols // 2, dtype=torch.uint8, device=dev),
               torch.empty(rows, cols // group, dtype=torch.int16, device=dev),
               torch.empty(rows, cols // group, dtype=torch.uint8, device=dev),
               torch.empty(rows, cols, dtype=torch.float32, device=dev) if want_W0 else None)
    codes, scale, zero, W0 = out
    _check(LIB.awsrc_backbone_rtn(_ptr(W), _dtype_code(W), rows, cols, group, _ptr(codes), _ptr(scale),
                                  _ptr(zero), _ptr(W0), _stream(stream)))
    return codes, scale, zero, W0


def encode_workspace_bytes(p: awsrc_params, W: torch.Tensor, d_mode: int) -> int:
    rows, cols = W.shape
    n = ctypes.c_size_t(0)
    _check(LIB.awsrc_encode_tiles(ctypes.byref(p), None, _dtype_code(W), None, rows, cols, None, d_mode,
                                  None, None, None, None, None, None, ctypes.byref(n), None))
    return n.value


SDQ_BLOCK = 256


def awsrc_sdq_encode(scale_f16: torch.Tensor, stream=None):
    """SDQ of fp16 group scales (int16 bit patterns, any shape, row-major):
    returns (codes int8 [n], block mean fp32 [nb], block step fp32 [nb])."""
    _dev(scale_f16)
    n = scale_f16.numel()
    nb = (n + SDQ_BLOCK - 1) // SDQ_BLOCK
    dev = scale_f16.device
    codes = torch.empty(n, dtype=torch.int8, device=dev)
    mean = torch.empty(nb, dtype=torch.float32, device=dev)
    step = torch.empty(nb, dtype=torch.float32, device=dev)
    _check(LIB.awsrc_sdq_encode(_ptr(scale_f16), n, _ptr(codes), _ptr(mean), _ptr(step), _stream(stream)))
    return codes, mean, step


def awsrc_backbone_sdq_dequant(codes: torch.Tensor, zero: torch.Tensor, sdq, group: int = 128,
                               out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """W0 [rows, cols] fp32 of the RTN-INT4-SDQ backbone (sdq = awsrc_sdq_encode's result)."""
    sc, mean, step = sdq
    _dev(codes, zero, sc, mean, step)
    rows, cols = codes.shape[0], codes.shape[1] * 2
    if out is None:
        out = torch.empty(rows, cols, dtype=torch.float32, device=codes.device)
    _check(LIB.awsrc_backbone_sdq_dequant(_ptr(codes), _ptr(zero), _ptr(sc), _ptr(mean), _ptr(step), rows, cols,
                                          group, _ptr(out), _stream(stream)))
    return out


def awsrc_encode_tiles(p: awsrc_params, W: torch.Tensor, W0: torch.Tensor, d: torch.Tensor,
                       want_alpha: bool = False, out: Optional[Dict[str, torch.Tensor]] = None,
                       workspace: Optional[torch.Tensor] = None, stream=None) -> Dict[str, torch.Tensor]:
    """Per-tile best seed, codes, fp16 scale bits, fp64 gain (and fp32 alpha*)."""
    _dev(W, W0, d)
    rows, cols = W.shape
    d_mode = AWSRC_D_PER_COL if d.dim() == 1 else AWSRC_D_PER_ELEM
    T = rows * cols // p.C
    dev = W.device
    if out is None:
        out = {"seed": torch.empty(T, dtype=torch.int16, device=dev),
               "codes": torch.empty(T, p.P, dtype=torch.int8, device=dev),
               "scale": torch.empty(T, dtype=torch.int16, device=dev),
               "gain": torch.empty(T, dtype=torch.float64, device=dev),
               "alpha": torch.empty(T, p.P, dtype=torch.float32, device=dev) if want_alpha else None}
    nbytes = encode_workspace_bytes(p, W, d_mode)
    if workspace is None or workspace.numel() < nbytes:
        workspace = _workspace(nbytes, dev)
    n = ctypes.c_size_t(workspace.numel())
    _check(LIB.awsrc_encode_tiles(ctypes.byref(p), _ptr(W), _dtype_code(W), _ptr(W0), rows, cols, _ptr(d),
                                  d_mode, _ptr(out["seed"]), _ptr(out["codes"]), _ptr(out["scale"]),
                                  _ptr(out["gain"]), _ptr(out.get("alpha")), _ptr(workspace),
                                  ctypes.byref(n), _stream(stream)))
    out["workspace"] = workspace
    return out


def _ptr_array(ts):
    return (ctypes.c_void_p * len(ts))(*[t.data_ptr() for t in ts])


def encode_modules_workspace_bytes(p: awsrc_params, shapes: Sequence[Tuple[int, int]], w_dtype: int,
                                   d_mode: int) -> int:
    n = ctypes.c_size_t(0)
    rows = _i64arr([s[0] for s in shapes])
    cols = _i64arr([s[1] for s in shapes])
    _check(LIB.awsrc_encode_modules(ctypes.byref(p), len(shapes), None, w_dtype, None, None, d_mode, rows, cols,
                                    None, None, None, None, None, None, ctypes.byref(n), None))
    return n.value


def awsrc_encode_modules(p: awsrc_params, W_list: Sequence[torch.Tensor], W0_list: Sequence[torch.Tensor],
                         d_list: Sequence[torch.Tensor], want_alpha: bool = False,
                         out: Optional[Dict[str, torch.Tensor]] = None, workspace: Optional[torch.Tensor] = None,
                         stream=None) -> Dict[str, torch.Tensor]:
    """awsrc_encode_tiles over several modules in one call; outputs
    concatenated in module order."""
    _dev(*W_list, *W0_list, *d_list)
    shapes = [tuple(w.shape) for w in W_list]
    dts = {_dtype_code(w) for w in W_list}
    if len(dts) != 1:
        raise TypeError("all W must share one dtype")
    w_dtype = dts.pop()
    modes = {AWSRC_D_PER_COL if d.dim() == 1 else AWSRC_D_PER_ELEM for d in d_list}
    if len(modes) != 1:
        raise TypeError("all d must be per column or all per element")
    d_mode = modes.pop()
    T = sum(r * c // p.C for r, c in shapes)
    dev = W_list[0].device
    if out is None:
        out = {"seed": torch.empty(T, dtype=torch.int16, device=dev),
               "codes": torch.empty(T, p.P, dtype=torch.int8, device=dev),
               "scale": torch.empty(T, dtype=torch.int16, device=dev),
               "gain": torch.empty(T, dtype=torch.float64, device=dev),
               "alpha": torch.empty(T, p.P, dtype=torch.float32, device=dev) if want_alpha else None}
    nbytes = encode_modules_workspace_bytes(p, shapes, w_dtype, d_mode)
    if workspace is None or workspace.numel() < nbytes:
        workspace = _workspace(nbytes, dev)
    n = ctypes.c_size_t(workspace.numel())
    rows = _i64arr([s[0] for s in shapes])
    cols = _i64arr([s[1] for s in shapes])
    _check(LIB.awsrc_encode_modules(ctypes.byref(p), len(shapes), _ptr_array(W_list), w_dtype, _ptr_array(W0_list),
                                    _ptr_array(d_list), d_mode, rows, cols, _ptr(out["seed"]), _ptr(out["codes"]),
                                    _ptr(out["scale"]), _ptr(out["gain"]), _ptr(out.get("alpha")), _ptr(workspace),
                                    ctypes.byref(n), _stream(stream)))
    out["workspace"] = workspace
    return out


def awsrc_encode_screen_lists(p: awsrc_params, shapes: Sequence[Tuple[int, int]], d_mode: int,
                              workspace: torch.Tensor, stream=None):
    """The fp32 screen's kept lists of the last encode with this workspace:
    (gain f32 [T, nsplit, 2], seed word int32 [T, nsplit, 2]: seed in bits
    0-15, bit 16 set for a candidate whose rounding was on a knife edge)."""
    rows = _i64arr([s[0] for s in shapes])
    cols = _i64arr([s[1] for s in shapes])
    ns = ctypes.c_int32(0)
    _check(LIB.awsrc_encode_screen_lists(ctypes.byref(p), len(shapes), rows, cols, d_mode, _ptr(workspace), None,
                                         None, ctypes.byref(ns), _stream(stream)))
    T = sum(r * c // p.C for r, c in shapes)
    g = torch.empty(T, ns.value, 2, dtype=torch.float32, device=workspace.device)
    sd = torch.empty(T, ns.value, 2, dtype=torch.int32, device=workspace.device)
    _check(LIB.awsrc_encode_screen_lists(ctypes.byref(p), len(shapes), rows, cols, d_mode, _ptr(workspace), _ptr(g),
                                         _ptr(sd), ctypes.byref(ns), _stream(stream)))
    return g, sd


def awsrc_encode_noalloc_max_bytes() -> int:
    return int(LIB.awsrc_encode_noalloc_max_bytes())


def awsrc_encode_tiles_noalloc(p: awsrc_params, W: torch.Tensor, W0: torch.Tensor, d: torch.Tensor,
                               out: Dict[str, torch.Tensor], stream=None) -> Dict[str, torch.Tensor]:
    """awsrc_encode_tiles into caller-provided outputs (keys seed, codes,
    scale, gain, optional alpha), with the library's fixed scratch array
    instead of a workspace: allocates nothing."""
    _dev(W, W0, d, *[v for v in out.values() if isinstance(v, torch.Tensor)])
    rows, cols = W.shape
    d_mode = AWSRC_D_PER_COL if d.dim() == 1 else AWSRC_D_PER_ELEM
    _check(LIB.awsrc_encode_tiles_noalloc(ctypes.byref(p), _ptr(W), _dtype_code(W), _ptr(W0), rows, cols, _ptr(d),
                                          d_mode, _ptr(out["seed"]), _ptr(out["codes"]), _ptr(out["scale"]),
                                          _ptr(out["gain"]), _ptr(out.get("alpha")), _stream(stream)))
    return out


def awsrc_encode_scored(out: Dict[str, torch.Tensor], stream=None) -> int:
    """Candidates scored in full by the last awsrc_encode_tiles call that filled `out`."""
    v = ctypes.c_uint64(0)
    _check(LIB.awsrc_encode_scored(_ptr(out["workspace"]), ctypes.byref(v), _stream(stream)))
    return int(v.value)


def _i64arr(v: Sequence[int]):
    return (ctypes.c_int64 * len(v))(*[int(x) for x in v])


def awsrc_rank_prefix(p: awsrc_params, modules: Sequence[Tuple[int, int]], mode: int, bpw: float,
                      seed: torch.Tensor, codes: torch.Tensor, scale: torch.Tensor, gain: torch.Tensor,
                      stream_cap: Optional[int] = None, out: Optional[torch.Tensor] = None,
                      workspace: Optional[torch.Tensor] = None, stream=None):
    """Rank and serialize; returns (stream bytes tensor [stream_len], K, n_eligible)."""
    _dev(seed, codes, scale, gain)
    rows = _i64arr([m[0] for m in modules])
    cols = _i64arr([m[1] for m in modules])
    n = ctypes.c_size_t(0)
    slen, K, ne = ctypes.c_uint64(0), ctypes.c_int64(0), ctypes.c_int64(0)
    _check(LIB.awsrc_rank_prefix(ctypes.byref(p), len(modules), rows, cols, mode, bpw, None, None, None, None,
                                 None, 0, ctypes.byref(slen), ctypes.byref(K), None, None, ctypes.byref(n), None))
    dev = gain.device
    if workspace is None or workspace.numel() < n.value:
        workspace = _workspace(n.value, dev)
    if out is None:
        if stream_cap is None:
            T = sum(r * c // p.C for r, c in modules)
            L = awsrc_record_bytes(p, T)
            N = sum(r * c for r, c in modules)
            if mode == AWSRC_MODE_GLOBAL:
                cap_rec = max(0, (awsrc_budget_bytes(bpw, N) - awsrc_header_bytes(len(modules))) // L)
            else:
                cap_rec = sum(awsrc_budget_bytes(bpw, r * c) // L for r, c in modules)
            stream_cap = awsrc_header_bytes(len(modules)) + min(cap_rec, T) * L
        out = torch.empty(int(stream_cap), dtype=torch.uint8, device=dev)
    cap = out.numel() if stream_cap is None else min(int(stream_cap), out.numel())
    n = ctypes.c_size_t(workspace.numel())
    _check(LIB.awsrc_rank_prefix(ctypes.byref(p), len(modules), rows, cols, mode, bpw, _ptr(seed), _ptr(codes),
                                 _ptr(scale), _ptr(gain), _ptr(out), cap, ctypes.byref(slen),
                                 ctypes.byref(K), ctypes.byref(ne), _ptr(workspace), ctypes.byref(n),
                                 _stream(stream)))
    return out[: slen.value], K.value, ne.value


def _decode_args(stream_bytes, W0_list, stream_len):
    _dev(stream_bytes, *W0_list)
    if stream_len is None:
        stream_len = stream_bytes.numel()
    dt = {_dtype_code(w) for w in W0_list}
    if len(dt) != 1:
        raise TypeError("all W0 must share one dtype")
    rows = _i64arr([w.shape[0] for w in W0_list])
    cols = _i64arr([w.shape[1] for w in W0_list])
    ptrs = (ctypes.c_void_p * len(W0_list))(*[w.data_ptr() for w in W0_list])
    return stream_len, rows, cols, ptrs, dt.pop()


def awsrc_decode_add(stream_bytes: torch.Tensor, W0_list: List[torch.Tensor], stream_len: Optional[int] = None,
                     workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    """In-place W0 += B_s alpha_hat for every record of the stream (or of its prefix)."""
    stream_len, rows, cols, ptrs, dt = _decode_args(stream_bytes, W0_list, stream_len)
    n = ctypes.c_size_t(0)
    st = _stream(stream)
    _check(LIB.awsrc_decode_add(_ptr(stream_bytes), stream_len, len(W0_list), ptrs, rows, cols, dt,
                                None, ctypes.byref(n), st))
    if workspace is None or workspace.numel() < n.value:
        workspace = _workspace(n.value, stream_bytes.device)
    n = ctypes.c_size_t(workspace.numel())
    _check(LIB.awsrc_decode_add(_ptr(stream_bytes), stream_len, len(W0_list), ptrs, rows, cols, dt,
                                _ptr(workspace), ctypes.byref(n), st))


def awsrc_decode_prepare(stream_bytes: torch.Tensor, W0_list: List[torch.Tensor], stream_len: Optional[int] = None,
                         workspace: Optional[torch.Tensor] = None, stream=None):
    """Validate a stream and build its decode tables; returns (plan, workspace).
    Keep both (and the stream bytes) alive while the plan is applied.  A
    workspace passed in (e.g. the one a previous plan used, once that plan is
    no longer needed) is used directly when it is large enough, which saves
    the size query's header read."""
    stream_len, rows, cols, ptrs, dt = _decode_args(stream_bytes, W0_list, stream_len)
    st = _stream(stream)
    plan = awsrc_decode_plan()
    if workspace is not None:
        n = ctypes.c_size_t(workspace.numel())
        rc = LIB.awsrc_decode_prepare(_ptr(stream_bytes), stream_len, len(W0_list), ptrs, rows, cols, dt,
                                      ctypes.byref(plan), _ptr(workspace), ctypes.byref(n), st)
        if rc != AWSRC_ENOSPC:
            _check(rc)
            return plan, workspace
    n = ctypes.c_size_t(0)
    _check(LIB.awsrc_decode_prepare(_ptr(stream_bytes), stream_len, len(W0_list), ptrs, rows, cols, dt, None,
                                    None, ctypes.byref(n), st))
    workspace = _workspace(n.value, stream_bytes.device)
    n = ctypes.c_size_t(workspace.numel())
    _check(LIB.awsrc_decode_prepare(_ptr(stream_bytes), stream_len, len(W0_list), ptrs, rows, cols, dt,
                                    ctypes.byref(plan), _ptr(workspace), ctypes.byref(n), st))
    return plan, workspace


def awsrc_decode_apply(plan: awsrc_decode_plan, stream=None) -> None:
    """One asynchronous launch adding every record of a prepared stream onto W0."""
    _check(LIB.awsrc_decode_apply(ctypes.byref(plan), _stream(stream)))


def awsrc_reconstruct_bf16(plan: awsrc_decode_plan, backbones: Sequence[Tuple[torch.Tensor, torch.Tensor,
                                                                               torch.Tensor]],
                           group: int = 128, stream=None) -> None:
    """Dense bf16(W0 + R_hat) into the bf16 buffers the plan was prepared on;
    `backbones` holds each module's (codes, scale, zero) as awsrc_backbone_rtn
    returns them."""
    if len(backbones) != plan.n_modules:
        raise ValueError(f"{len(backbones)} backbones for a plan of {plan.n_modules} modules")
    for bb in backbones:
        _dev(*bb)
    arr = [(ctypes.c_void_p * len(backbones))(*[bb[k].data_ptr() for bb in backbones]) for k in range(3)]
    _check(LIB.awsrc_reconstruct_bf16(ctypes.byref(plan), group, arr[0], arr[1], arr[2], _stream(stream)))


def awsrc_reconstruct_bf16_prefixes(plan: awsrc_decode_plan, K_out: Sequence[int],
                                    outs: Sequence[Sequence[torch.Tensor]],
                                    backbones: Sequence[Tuple[torch.Tensor, torch.Tensor, torch.Tensor]],
                                    group: int = 128, stream=None) -> None:
    """Dense bf16(W0 + R_hat of the first K_out[o] records) into outs[o] (one
    bf16 tensor per module) for every o, in one pass over the backbone."""
    n = plan.n_modules
    if len(backbones) != n or len(outs) != len(K_out) or any(len(o) != n for o in outs):
        raise ValueError("need one backbone and, per prefix, one target per module")
    for bb in backbones:
        _dev(*bb)
    for o in outs:
        _dev(*o)
        if any(t.dtype != torch.bfloat16 for t in o):
            raise TypeError("targets must be bf16")
    arr = [(ctypes.c_void_p * n)(*[bb[k].data_ptr() for bb in backbones]) for k in range(3)]
    optr = (ctypes.c_void_p * (n * len(outs)))(*[t.data_ptr() for o in outs for t in o])
    _check(LIB.awsrc_reconstruct_bf16_prefixes(ctypes.byref(plan), len(K_out), _i64arr(list(K_out)), optr, group,
                                               arr[0], arr[1], arr[2], _stream(stream)))


def awsrc_reconstruct_bf16_sdq(plan: awsrc_decode_plan,
                               backbones: Sequence[Tuple[torch.Tensor, torch.Tensor, torch.Tensor, torch.Tensor,
                                                         torch.Tensor]],
                               K_out: Optional[Sequence[int]] = None,
                               outs: Optional[Sequence[Sequence[torch.Tensor]]] = None,
                               group: int = 128, stream=None) -> None:
    """Dense bf16 repaired weights on the RTN-INT4-SDQ backbone: `backbones`
    holds each module's (codes, zero, sdq_code, sdq_mean, sdq_step), the RTN
    codes and zero points with awsrc_sdq_encode's outputs for its scales.
    Without K_out / outs: into the bf16 buffers the plan was prepared on, every
    record; else outs[o] receives the first K_out[o] records' prefix."""
    n = plan.n_modules
    if len(backbones) != n:
        raise ValueError(f"{len(backbones)} backbones for a plan of {n} modules")
    for bb in backbones:
        _dev(*bb)
    if (K_out is None) != (outs is None):
        raise ValueError("K_out and outs go together")
    arr = [(ctypes.c_void_p * n)(*[bb[k].data_ptr() for bb in backbones]) for k in range(5)]
    if outs is None:
        n_out, kp, optr = 0, None, None
    else:
        if len(outs) != len(K_out) or any(len(o) != n for o in outs):
            raise ValueError("need, per prefix, one target per module")
        for o in outs:
            _dev(*o)
            if any(t.dtype != torch.bfloat16 for t in o):
                raise TypeError("targets must be bf16")
        n_out, kp = len(K_out), _i64arr(list(K_out))
        optr = (ctypes.c_void_p * (n * n_out))(*[t.data_ptr() for o in outs for t in o])
    _check(LIB.awsrc_reconstruct_bf16_sdq(ctypes.byref(plan), n_out, kp, optr, group, arr[0], arr[2], arr[3], arr[4],
                                          arr[1], _stream(stream)))
