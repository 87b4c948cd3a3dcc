"""MI355X (gfx950) fused BitLinear: Python binding of ``libmmf.so``.

The forward pass of the BitLinear layer of "Scalable MatMul-free Language
Modeling" (arXiv 2406.02528; Algorithm 1 with bias 0): RMSNorm, per-token
absmax int8 quantisation, ternary accumulation with int32 sums and
dequantisation.  Every step runs in the HIP kernels of ``libmmf.so``; this
module only checks tensor shapes, dtypes and devices and passes raw pointers
and the current HIP stream through the C ABI declared in ``include/mmf.h``.
PyTorch is used for device memory and streams only.

Also the GLU channel mixer's gated up-projection, the MLGRU token mixer
(input projections with gate activations, the recurrence, the whole mixer),
and the training forward and backward of the layer.

Functions carry the names of the C entry points.  There is no fallback: if
the library is not built, importing this package raises ``ImportError``.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmmf.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; g.build()'` "
        "(hipcc --offload-arch=gfx950); there is no CPU fallback")

_lib = ctypes.CDLL(LIB_PATH)

MMF_OK = 0
MMF_PATH_AUTO, MMF_PATH_GEMV, MMF_PATH_GEMM = 0, 1, 2

_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_SZ = ctypes.c_size_t

_SIGNATURES = {
    "mmf_status_string": ([ctypes.c_int], ctypes.c_char_p),
    "mmf_version": ([], ctypes.c_int),
    "mmf_packed_weight_bytes": ([_I64, _I64], _SZ),
    "mmf_ternarize_weights": ([_P, _I64, _I64, _P, _P, _P], ctypes.c_int),
    "mmf_act_quant": ([_P, _P, _P, _P, _I64, _I64, _P], ctypes.c_int),
    "mmf_act_quant_f32": ([_P, _P, _P, _P, _I64, _I64, _P], ctypes.c_int),
    "mmf_act_quant_ex": ([_P, ctypes.c_int, _P, _P, _P, _P, _I64, _I64, _P], ctypes.c_int),
    "mmf_bitlinear_fwd": ([_P, _P, _P, _P, _P, _I64, _I64, _I64, _P], ctypes.c_int),
    "mmf_bitlinear_fwd_f32": ([_P, _P, _P, _P, _P, _I64, _I64, _I64, _P], ctypes.c_int),
    "mmf_bitlinear_workspace_bytes": ([_I64, _I64], _SZ),
    "mmf_bitlinear_fwd_ws": ([_P, ctypes.c_int, _P, _P, _P, _P, _I64, _I64, _I64, _P, _SZ, _P],
                             ctypes.c_int),
    "mmf_bitlinear_noalloc_max_bytes": ([], _SZ),
    "mmf_bitlinear_fwd_noalloc": ([_P, ctypes.c_int, _P, _P, _P, _P, _I64, _I64, _I64, _P],
                                  ctypes.c_int),
    "mmf_ternary_gemm_dequant": ([_P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _P], ctypes.c_int),
    "mmf_ternary_gemm_i32": ([_P, _P, _P, _I64, _I64, _I64, _P], ctypes.c_int),
    "mmf_set_path": ([ctypes.c_int], ctypes.c_int),
    "mmf_prefill_tile_plan": ([ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int, ctypes.c_int],
                              ctypes.c_int),
    "mmf_glu_pack": ([_P, _P, _I64, _I64, _P, _P], ctypes.c_int),
    "mmf_glu_fwd": ([_P, _P, _P, _P, _P, _I64, _I64, _I64, _P], ctypes.c_int),
    "mmf_glu_fwd_f32": ([_P, _P, _P, _P, _P, _I64, _I64, _I64, _P], ctypes.c_int),
    "mmf_glu_fwd_ws": ([_P, ctypes.c_int, _P, _P, _P, _P, _I64, _I64, _I64, _P, _SZ, _P],
                       ctypes.c_int),
    "mmf_ternary_gemm_glu": ([_P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _P], ctypes.c_int),
    "mmf_bitlinear_fwd_bias": ([_P, ctypes.c_int, _P, _P, _P, _P, _P, _I64, _I64, _I64, _P],
                               ctypes.c_int),
    "mmf_mlgru_proj_workspace_bytes": ([_I64, _I64, _I64], _SZ),
    "mmf_mlgru_proj": ([_P, ctypes.c_int, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _P, _SZ, _P],
                       ctypes.c_int),
    "mmf_mlgru_proj_q": ([_P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _P], ctypes.c_int),
    "mmf_mlgru_scan_workspace_bytes": ([_I64, _I64, _I64], _SZ),
    "mmf_mlgru_scan": ([_P, _P, _P, _P, _I64, _I64, _I64, _P, _SZ, _P], ctypes.c_int),
    "mmf_mlgru_workspace_bytes": ([_I64, _I64, _I64], _SZ),
    "mmf_bitlinear_train_workspace_bytes": ([_I64, _I64, _I64], _SZ),
    "mmf_bitlinear_train_fwd": ([_P, ctypes.c_int, _P, _P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64,
                                 _I64, _P, _SZ, _P], ctypes.c_int),
    "mmf_bitlinear_bwd_workspace_bytes": ([_I64, _I64, _I64], _SZ),
    "mmf_bitlinear_bwd": ([_P, _P, ctypes.c_int, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64,
                           _I64, _P, _SZ, _P], ctypes.c_int),
    "mmf_mlgru_fwd": ([_P, ctypes.c_int, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                       _I64, _I64, _I64, _P, _SZ, _P], ctypes.c_int),
}
for _name, (_args, _res) in _SIGNATURES.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = _res


class MMFError(RuntimeError):
    pass


def _check(status: int) -> None:
    if status != MMF_OK:
        raise MMFError(_lib.mmf_status_string(status).decode())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _ptr(t: torch.Tensor | None) -> ctypes.c_void_p:
    return ctypes.c_void_p(0 if t is None else t.data_ptr())


def _need(t: torch.Tensor, name: str, dtype, shape) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a HIP device")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _x_kind(x: torch.Tensor) -> bool:
    """True for float32 activations, False for bfloat16."""
    if x.dtype == torch.float32:
        return True
    if x.dtype == torch.bfloat16:
        return False
    raise TypeError(f"x must be bfloat16 or float32, got {x.dtype}")


def mmf_version() -> int:
    return int(_lib.mmf_version())


def mmf_status_string(status: int) -> str:
    return _lib.mmf_status_string(int(status)).decode()


def mmf_packed_weight_bytes(N: int, K: int) -> int:
    return int(_lib.mmf_packed_weight_bytes(N, K))


def mmf_set_path(path: int) -> int:
    prev = int(_lib.mmf_set_path(int(path)))
    if prev < 0:
        raise ValueError(f"unknown path {path}")
    return prev


MMF_EPILOGUE_DEQUANT, MMF_EPILOGUE_RAW_I32, MMF_EPILOGUE_GLU, MMF_EPILOGUE_AFFINE = 0, 1, 2, 3
TILE_PLANS = ("128x512", "128x256_paired", "64x512", "64x256", "256x256")


def mmf_prefill_tile_plan(M: int, K: int, N: int, epilogue: int = MMF_EPILOGUE_DEQUANT, cus: int = 256) -> str:
    """The prefill contraction's tile plan for M x K x N on `cus` compute
    units (host only), as a name from TILE_PLANS."""
    r = int(_lib.mmf_prefill_tile_plan(M, K, N, epilogue, cus))
    _check(-r if r < 0 else 0)
    return TILE_PLANS[r]


def mmf_ternarize_weights(W: torch.Tensor, Wpacked: torch.Tensor, w_scale: torch.Tensor,
                          stream=None) -> None:
    """W float32 [N][K] -> Wpacked int32 [K/16][N] (uint32 bit patterns), w_scale float32 [1]."""
    N, K = W.shape
    _need(W, "W", torch.float32, (N, K))
    _need(Wpacked, "Wpacked", torch.int32, (K // 16, N))
    _need(w_scale, "w_scale", torch.float32, (1,))
    _check(_lib.mmf_ternarize_weights(_ptr(W), N, K, _ptr(Wpacked), _ptr(w_scale), _stream(stream)))


def mmf_act_quant(x: torch.Tensor, gamma: torch.Tensor | None, q: torch.Tensor,
                  a_scale: torch.Tensor, q_rowsum: torch.Tensor | None = None,
                  stream=None) -> None:
    """x bf16/f32 [M][K], gamma f32 [K] or None -> q int8 [M][K], a_scale f32 [M], q_rowsum i32 [M]."""
    M, K = x.shape
    is_f32 = _x_kind(x)
    _need(x, "x", x.dtype, (M, K))
    if gamma is not None:
        _need(gamma, "gamma", torch.float32, (K,))
    _need(q, "q", torch.int8, (M, K))
    _need(a_scale, "a_scale", torch.float32, (M,))
    if q_rowsum is not None:
        _need(q_rowsum, "q_rowsum", torch.int32, (M,))
        _check(_lib.mmf_act_quant_ex(_ptr(x), int(is_f32), _ptr(gamma), _ptr(q), _ptr(a_scale),
                                     _ptr(q_rowsum), M, K, _stream(stream)))
        return
    fn = _lib.mmf_act_quant_f32 if is_f32 else _lib.mmf_act_quant
    _check(fn(_ptr(x), _ptr(gamma), _ptr(q), _ptr(a_scale), M, K, _stream(stream)))


def mmf_act_quant_ex(x: torch.Tensor, gamma: torch.Tensor | None, q: torch.Tensor,
                     a_scale: torch.Tensor, q_rowsum: torch.Tensor | None, stream=None) -> None:
    """mmf_act_quant with the row sums q_rowsum i32 [M] (None: not written)."""
    mmf_act_quant(x, gamma, q, a_scale, q_rowsum, stream)


def mmf_bitlinear_fwd(x: torch.Tensor, gamma: torch.Tensor | None, Wpacked: torch.Tensor,
                      w_scale: torch.Tensor, y: torch.Tensor, stream=None) -> None:
    """The fused forward: y f32 [M][N] from x bf16/f32 [M][K] and packed weights [K/16][N]."""
    M, K = x.shape
    N = Wpacked.shape[1]
    is_f32 = _x_kind(x)
    _need(x, "x", x.dtype, (M, K))
    if gamma is not None:
        _need(gamma, "gamma", torch.float32, (K,))
    _need(Wpacked, "Wpacked", torch.int32, (K // 16, N))
    _need(w_scale, "w_scale", torch.float32, (1,))
    _need(y, "y", torch.float32, (M, N))
    fn = _lib.mmf_bitlinear_fwd_f32 if is_f32 else _lib.mmf_bitlinear_fwd
    _check(fn(_ptr(x), _ptr(gamma), _ptr(Wpacked), _ptr(w_scale), _ptr(y), M, K, N,
              _stream(stream)))


def mmf_bitlinear_workspace_bytes(M: int, K: int) -> int:
    return int(_lib.mmf_bitlinear_workspace_bytes(M, K))


def mmf_bitlinear_fwd_ws(x: torch.Tensor, gamma: torch.Tensor | None, Wpacked: torch.Tensor,
                         w_scale: torch.Tensor, y: torch.Tensor, workspace: torch.Tensor,
                         stream=None) -> None:
    """The fused forward with caller scratch (a uint8 device tensor)."""
    M, K = x.shape
    N = Wpacked.shape[1]
    is_f32 = _x_kind(x)
    _need(x, "x", x.dtype, (M, K))
    if gamma is not None:
        _need(gamma, "gamma", torch.float32, (K,))
    _need(Wpacked, "Wpacked", torch.int32, (K // 16, N))
    _need(w_scale, "w_scale", torch.float32, (1,))
    _need(y, "y", torch.float32, (M, N))
    _need(workspace, "workspace", torch.uint8, (workspace.numel(),))
    _check(_lib.mmf_bitlinear_fwd_ws(_ptr(x), int(is_f32), _ptr(gamma), _ptr(Wpacked),
                                     _ptr(w_scale), _ptr(y), M, K, N, _ptr(workspace),
                                     workspace.numel(), _stream(stream)))


def mmf_bitlinear_noalloc_max_bytes() -> int:
    return int(_lib.mmf_bitlinear_noalloc_max_bytes())


def mmf_bitlinear_fwd_noalloc(x: torch.Tensor, gamma: torch.Tensor | None, Wpacked: torch.Tensor,
                              w_scale: torch.Tensor, y: torch.Tensor, stream=None) -> None:
    """The fused forward with the library's static device scratch (allocates nothing)."""
    M, K = x.shape
    N = Wpacked.shape[1]
    is_f32 = _x_kind(x)
    _need(x, "x", x.dtype, (M, K))
    if gamma is not None:
        _need(gamma, "gamma", torch.float32, (K,))
    _need(Wpacked, "Wpacked", torch.int32, (K // 16, N))
    _need(w_scale, "w_scale", torch.float32, (1,))
    _need(y, "y", torch.float32, (M, N))
    _check(_lib.mmf_bitlinear_fwd_noalloc(_ptr(x), int(is_f32), _ptr(gamma), _ptr(Wpacked),
                                          _ptr(w_scale), _ptr(y), M, K, N, _stream(stream)))


def mmf_ternary_gemm_dequant(q: torch.Tensor, a_scale: torch.Tensor, q_rowsum: torch.Tensor,
                             Wpacked: torch.Tensor, w_scale: torch.Tensor, y: torch.Tensor,
                             stream=None) -> None:
    """Contraction + dequant from quantised activations (the forward after act-quant)."""
    M, K = q.shape
    N = Wpacked.shape[1]
    _need(q, "q", torch.int8, (M, K))
    _need(a_scale, "a_scale", torch.float32, (M,))
    _need(q_rowsum, "q_rowsum", torch.int32, (M,))
    _need(Wpacked, "Wpacked", torch.int32, (K // 16, N))
    _need(w_scale, "w_scale", torch.float32, (1,))
    _need(y, "y", torch.float32, (M, N))
    _check(_lib.mmf_ternary_gemm_dequant(_ptr(q), _ptr(a_scale), _ptr(q_rowsum), _ptr(Wpacked),
                                         _ptr(w_scale), _ptr(y), M, K, N, _stream(stream)))


def mmf_ternary_gemm_i32(q: torch.Tensor, Wpacked: torch.Tensor, acc: torch.Tensor,
                         stream=None) -> None:
    """Raw int32 ternary sums acc [M][N] from q int8 [M][K] and packed weights."""
    M, K = q.shape
    N = Wpacked.shape[1]
    _need(q, "q", torch.int8, (M, K))
    _need(Wpacked, "Wpacked", torch.int32, (K // 16, N))
    _need(acc, "acc", torch.int32, (M, N))
    _check(_lib.mmf_ternary_gemm_i32(_ptr(q), _ptr(Wpacked), _ptr(acc), M, K, N, _stream(stream)))


def mmf_glu_pack(Wg_packed: torch.Tensor, Wu_packed: torch.Tensor, Wgu_packed: torch.Tensor,
                 stream=None) -> None:
    """Interleave the packed gate and up projections [K/16][L] into [K/16][2L]
    (16-column blocks of gate and up in turn); L % 16 == 0."""
    J, L = Wg_packed.shape
    _need(Wg_packed, "Wg_packed", torch.int32, (J, L))
    _need(Wu_packed, "Wu_packed", torch.int32, (J, L))
    _need(Wgu_packed, "Wgu_packed", torch.int32, (J, 2 * L))
    _check(_lib.mmf_glu_pack(_ptr(Wg_packed), _ptr(Wu_packed), L, 16 * J, _ptr(Wgu_packed),
                             _stream(stream)))


def _glu_args(x, gamma, Wgu_packed, w_scales, p):
    M, K = x.shape
    L = Wgu_packed.shape[1] // 2
    is_f32 = _x_kind(x)
    _need(x, "x", x.dtype, (M, K))
    if gamma is not None:
        _need(gamma, "gamma", torch.float32, (K,))
    _need(Wgu_packed, "Wgu_packed", torch.int32, (K // 16, 2 * L))
    _need(w_scales, "w_scales", torch.float32, (2,))
    _need(p, "p", torch.float32, (M, L))
    return M, K, L, is_f32


def mmf_glu_fwd(x: torch.Tensor, gamma: torch.Tensor | None, Wgu_packed: torch.Tensor,
                w_scales: torch.Tensor, p: torch.Tensor, stream=None) -> None:
    """GLU up-projections and gate: p f32 [M][L] = SiLU(g) * u from x bf16/f32
    [M][K], the interleaved packed weights [K/16][2L] and w_scales [gate, up]."""
    M, K, L, is_f32 = _glu_args(x, gamma, Wgu_packed, w_scales, p)
    fn = _lib.mmf_glu_fwd_f32 if is_f32 else _lib.mmf_glu_fwd
    _check(fn(_ptr(x), _ptr(gamma), _ptr(Wgu_packed), _ptr(w_scales), _ptr(p), M, K, L,
              _stream(stream)))


def mmf_glu_fwd_ws(x: torch.Tensor, gamma: torch.Tensor | None, Wgu_packed: torch.Tensor,
                   w_scales: torch.Tensor, p: torch.Tensor, workspace: torch.Tensor,
                   stream=None) -> None:
    """mmf_glu_fwd with caller scratch (uint8, mmf_bitlinear_workspace_bytes(M, K))."""
    M, K, L, is_f32 = _glu_args(x, gamma, Wgu_packed, w_scales, p)
    _need(workspace, "workspace", torch.uint8, (workspace.numel(),))
    _check(_lib.mmf_glu_fwd_ws(_ptr(x), int(is_f32), _ptr(gamma), _ptr(Wgu_packed),
                               _ptr(w_scales), _ptr(p), M, K, L, _ptr(workspace),
                               workspace.numel(), _stream(stream)))


def mmf_ternary_gemm_glu(q: torch.Tensor, a_scale: torch.Tensor, q_rowsum: torch.Tensor,
                         Wgu_packed: torch.Tensor, w_scales: torch.Tensor, p: torch.Tensor,
                         stream=None) -> None:
    """The GLU contraction and gate from quantised activations: p [M][L]."""
    M, K = q.shape
    L = Wgu_packed.shape[1] // 2
    _need(q, "q", torch.int8, (M, K))
    _need(a_scale, "a_scale", torch.float32, (M,))
    _need(q_rowsum, "q_rowsum", torch.int32, (M,))
    _need(Wgu_packed, "Wgu_packed", torch.int32, (K // 16, 2 * L))
    _need(w_scales, "w_scales", torch.float32, (2,))
    _need(p, "p", torch.float32, (M, L))
    _check(_lib.mmf_ternary_gemm_glu(_ptr(q), _ptr(a_scale), _ptr(q_rowsum), _ptr(Wgu_packed),
                                     _ptr(w_scales), _ptr(p), M, K, L, _stream(stream)))


def _ws_args(workspace: torch.Tensor | None):
    if workspace is None:
        return _ptr(None), 0
    _need(workspace, "workspace", torch.uint8, (workspace.numel(),))
    return _ptr(workspace), workspace.numel()


def mmf_bitlinear_fwd_bias(x: torch.Tensor, gamma: torch.Tensor | None, Wpacked: torch.Tensor,
                           w_scale: torch.Tensor, bias: torch.Tensor, y: torch.Tensor,
                           stream=None) -> None:
    """y f32 [M][N] = BitLinear(x) + bias [N] (N % 4 == 0)."""
    M, K = x.shape
    N = Wpacked.shape[1]
    is_f32 = _x_kind(x)
    _need(x, "x", x.dtype, (M, K))
    if gamma is not None:
        _need(gamma, "gamma", torch.float32, (K,))
    _need(Wpacked, "Wpacked", torch.int32, (K // 16, N))
    _need(w_scale, "w_scale", torch.float32, (1,))
    _need(bias, "bias", torch.float32, (N,))
    _need(y, "y", torch.float32, (M, N))
    _check(_lib.mmf_bitlinear_fwd_bias(_ptr(x), int(is_f32), _ptr(gamma), _ptr(Wpacked),
                                       _ptr(w_scale), _ptr(bias), _ptr(y), M, K, N,
                                       _stream(stream)))


def mmf_mlgru_proj_workspace_bytes(M: int, K: int, d: int) -> int:
    return int(_lib.mmf_mlgru_proj_workspace_bytes(M, K, d))


def mmf_mlgru_scan_workspace_bytes(B: int, T: int, d: int) -> int:
    return int(_lib.mmf_mlgru_scan_workspace_bytes(B, T, d))


def mmf_mlgru_workspace_bytes(B: int, T: int, d: int) -> int:
    return int(_lib.mmf_mlgru_workspace_bytes(B, T, d))


def mmf_mlgru_proj(x: torch.Tensor, gamma: torch.Tensor | None, Wfcg: torch.Tensor,
                   w_scales: torch.Tensor, bias: torch.Tensor | None, lb: torch.Tensor | None,
                   fcg: torch.Tensor, workspace: torch.Tensor | None = None, stream=None) -> None:
    """MLGRU input projections and gates: fcg f32 [M][3d] (f | c | g) from x
    bf16/f32 [M][K], Wfcg [K/16][3d], w_scales [3], bias [3d] or None, lb [d]
    or None."""
    M, K = x.shape
    d = Wfcg.shape[1] // 3
    is_f32 = _x_kind(x)
    _need(x, "x", x.dtype, (M, K))
    if gamma is not None:
        _need(gamma, "gamma", torch.float32, (K,))
    _need(Wfcg, "Wfcg", torch.int32, (K // 16, 3 * d))
    _need(w_scales, "w_scales", torch.float32, (3,))
    if bias is not None:
        _need(bias, "bias", torch.float32, (3 * d,))
    if lb is not None:
        _need(lb, "lb", torch.float32, (d,))
    _need(fcg, "fcg", torch.float32, (M, 3 * d))
    wp, wn = _ws_args(workspace)
    _check(_lib.mmf_mlgru_proj(_ptr(x), int(is_f32), _ptr(gamma), _ptr(Wfcg), _ptr(w_scales),
                               _ptr(bias), _ptr(lb), _ptr(fcg), M, K, d, wp, wn, _stream(stream)))


def mmf_mlgru_proj_q(q: torch.Tensor, a_scale: torch.Tensor, q_rowsum: torch.Tensor,
                     Wfcg: torch.Tensor, w_scales: torch.Tensor, bias: torch.Tensor | None,
                     lb: torch.Tensor | None, fcg: torch.Tensor, stream=None) -> None:
    """The MLGRU projection's contraction and gates from quantised activations."""
    M, K = q.shape
    d = Wfcg.shape[1] // 3
    _need(q, "q", torch.int8, (M, K))
    _need(a_scale, "a_scale", torch.float32, (M,))
    _need(q_rowsum, "q_rowsum", torch.int32, (M,))
    _need(Wfcg, "Wfcg", torch.int32, (K // 16, 3 * d))
    _need(w_scales, "w_scales", torch.float32, (3,))
    if bias is not None:
        _need(bias, "bias", torch.float32, (3 * d,))
    if lb is not None:
        _need(lb, "lb", torch.float32, (d,))
    _need(fcg, "fcg", torch.float32, (M, 3 * d))
    _check(_lib.mmf_mlgru_proj_q(_ptr(q), _ptr(a_scale), _ptr(q_rowsum), _ptr(Wfcg),
                                 _ptr(w_scales), _ptr(bias), _ptr(lb), _ptr(fcg), M, K, d,
                                 _stream(stream)))


def mmf_mlgru_scan(fcg: torch.Tensor, B: int, T: int, h0: torch.Tensor | None,
                   o_prime: torch.Tensor, h_last: torch.Tensor | None,
                   workspace: torch.Tensor | None = None, stream=None) -> None:
    """MLGRU recurrence and output gate over B sequences of T tokens (rows
    b*T + t): o_prime f32 [B*T][d], final state h_last [B][d] (may be h0)."""
    d = fcg.shape[1] // 3
    _need(fcg, "fcg", torch.float32, (B * T, 3 * d))
    if h0 is not None:
        _need(h0, "h0", torch.float32, (B, d))
    _need(o_prime, "o_prime", torch.float32, (B * T, d))
    if h_last is not None:
        _need(h_last, "h_last", torch.float32, (B, d))
    wp, wn = _ws_args(workspace)
    _check(_lib.mmf_mlgru_scan(_ptr(fcg), _ptr(h0), _ptr(o_prime), _ptr(h_last), B, T, d, wp, wn,
                               _stream(stream)))


def mmf_mlgru_fwd(x: torch.Tensor, B: int, T: int, gamma: torch.Tensor | None,
                  Wfcg: torch.Tensor, w_scales: torch.Tensor, bias: torch.Tensor | None,
                  lb: torch.Tensor | None, h0: torch.Tensor | None, h_last: torch.Tensor | None,
                  gamma_o: torch.Tensor | None, Wo: torch.Tensor, w_scale_o: torch.Tensor,
                  b_o: torch.Tensor | None, o: torch.Tensor,
                  workspace: torch.Tensor | None = None, stream=None) -> None:
    """The whole MLGRU token mixer: o f32 [B*T][d] from x bf16/f32 [B*T][d]."""
    d = Wo.shape[1]
    is_f32 = _x_kind(x)
    _need(x, "x", x.dtype, (B * T, d))
    for name, t, shape in (("gamma", gamma, (d,)), ("bias", bias, (3 * d,)), ("lb", lb, (d,)),
                           ("h0", h0, (B, d)), ("h_last", h_last, (B, d)),
                           ("gamma_o", gamma_o, (d,)), ("b_o", b_o, (d,))):
        if t is not None:
            _need(t, name, torch.float32, shape)
    _need(Wfcg, "Wfcg", torch.int32, (d // 16, 3 * d))
    _need(w_scales, "w_scales", torch.float32, (3,))
    _need(Wo, "Wo", torch.int32, (d // 16, d))
    _need(w_scale_o, "w_scale_o", torch.float32, (1,))
    _need(o, "o", torch.float32, (B * T, d))
    wp, wn = _ws_args(workspace)
    _check(_lib.mmf_mlgru_fwd(_ptr(x), int(is_f32), _ptr(gamma), _ptr(Wfcg), _ptr(w_scales),
                              _ptr(bias), _ptr(lb), _ptr(h0), _ptr(h_last), _ptr(gamma_o),
                              _ptr(Wo), _ptr(w_scale_o), _ptr(b_o), _ptr(o), B, T, d, wp, wn,
                              _stream(stream)))


def mmf_bitlinear_train_workspace_bytes(M: int, K: int, N: int) -> int:
    return int(_lib.mmf_bitlinear_train_workspace_bytes(M, K, N))


def mmf_bitlinear_bwd_workspace_bytes(M: int, K: int, N: int) -> int:
    return int(_lib.mmf_bitlinear_bwd_workspace_bytes(M, K, N))


def mmf_bitlinear_train_fwd(x: torch.Tensor, gamma: torch.Tensor | None, W: torch.Tensor,
                            bias: torch.Tensor | None, y: torch.Tensor, Wpacked: torch.Tensor,
                            w_scale: torch.Tensor, q: torch.Tensor, a_scale: torch.Tensor,
                            rstd: torch.Tensor | None, workspace: torch.Tensor | None = None,
                            stream=None) -> None:
    """Training forward from latent float32 weights W [N][K]: y [M][N] and the
    state the backward needs (Wpacked, w_scale, q, a_scale, rstd)."""
    M, K = x.shape
    N = W.shape[0]
    is_f32 = _x_kind(x)
    _need(x, "x", x.dtype, (M, K))
    if gamma is not None:
        _need(gamma, "gamma", torch.float32, (K,))
    _need(W, "W", torch.float32, (N, K))
    if bias is not None:
        _need(bias, "bias", torch.float32, (N,))
    _need(y, "y", torch.float32, (M, N))
    _need(Wpacked, "Wpacked", torch.int32, (K // 16, N))
    _need(w_scale, "w_scale", torch.float32, (1,))
    _need(q, "q", torch.int8, (M, K))
    _need(a_scale, "a_scale", torch.float32, (M,))
    if rstd is not None:
        _need(rstd, "rstd", torch.float32, (M,))
    wp, wn = _ws_args(workspace)
    _check(_lib.mmf_bitlinear_train_fwd(_ptr(x), int(is_f32), _ptr(gamma), _ptr(W), _ptr(bias), _ptr(y),
                                        _ptr(Wpacked), _ptr(w_scale), _ptr(q), _ptr(a_scale), _ptr(rstd),
                                        M, K, N, wp, wn, _stream(stream)))


def mmf_bitlinear_bwd(dO: torch.Tensor, x: torch.Tensor, gamma: torch.Tensor | None,
                      rstd: torch.Tensor, q: torch.Tensor, a_scale: torch.Tensor,
                      Wpacked: torch.Tensor, w_scale: torch.Tensor, dx: torch.Tensor,
                      dW: torch.Tensor, db: torch.Tensor | None, dgamma: torch.Tensor | None,
                      workspace: torch.Tensor | None = None, stream=None) -> None:
    """Backward: dx [M][K], dW [N][K], db [N], dgamma [K] (float32) from dO
    bf16 [M][N] and the training forward's saved state."""
    M, K = x.shape
    N = dO.shape[1]
    is_f32 = _x_kind(x)
    _need(dO, "dO", torch.bfloat16, (M, N))
    _need(x, "x", x.dtype, (M, K))
    if gamma is not None:
        _need(gamma, "gamma", torch.float32, (K,))
    _need(rstd, "rstd", torch.float32, (M,))
    _need(q, "q", torch.int8, (M, K))
    _need(a_scale, "a_scale", torch.float32, (M,))
    _need(Wpacked, "Wpacked", torch.int32, (K // 16, N))
    _need(w_scale, "w_scale", torch.float32, (1,))
    _need(dx, "dx", torch.float32, (M, K))
    _need(dW, "dW", torch.float32, (N, K))
    if db is not None:
        _need(db, "db", torch.float32, (N,))
    if dgamma is not None:
        _need(dgamma, "dgamma", torch.float32, (K,))
    wp, wn = _ws_args(workspace)
    _check(_lib.mmf_bitlinear_bwd(_ptr(dO), _ptr(x), int(is_f32), _ptr(gamma), _ptr(rstd), _ptr(q),
                                  _ptr(a_scale), _ptr(Wpacked), _ptr(w_scale), _ptr(dx), _ptr(dW),
                                  _ptr(db), _ptr(dgamma), M, K, N, wp, wn, _stream(stream)))


# ---------------------------------------------------------------------------
# allocating conveniences (outputs allocated with torch on the inputs' device)
# ---------------------------------------------------------------------------

def ternarize(W: torch.Tensor, stream=None):
    """Returns (Wpacked int32 [K/16][N], w_scale float32 [1])."""
    N, K = W.shape
    Wp = torch.empty((K // 16, N), dtype=torch.int32, device=W.device)
    ws = torch.empty((1,), dtype=torch.float32, device=W.device)
    mmf_ternarize_weights(W, Wp, ws, stream)
    return Wp, ws


def bitlinear(x: torch.Tensor, gamma: torch.Tensor | None, Wpacked: torch.Tensor,
              w_scale: torch.Tensor, stream=None) -> torch.Tensor:
    """Returns y float32 [M][N]."""
    y = torch.empty((x.shape[0], Wpacked.shape[1]), dtype=torch.float32, device=x.device)
    mmf_bitlinear_fwd(x, gamma, Wpacked, w_scale, y, stream)
    return y


def glu_pack(Wg_packed: torch.Tensor, Wu_packed: torch.Tensor, stream=None) -> torch.Tensor:
    """Returns the interleaved [K/16][2L] packed weights of a GLU."""
    J, L = Wg_packed.shape
    Wgu = torch.empty((J, 2 * L), dtype=torch.int32, device=Wg_packed.device)
    mmf_glu_pack(Wg_packed, Wu_packed, Wgu, stream)
    return Wgu


def glu(x: torch.Tensor, gamma: torch.Tensor | None, Wgu_packed: torch.Tensor,
        w_scales: torch.Tensor, stream=None) -> torch.Tensor:
    """Returns p float32 [M][L] = SiLU(g) * u."""
    p = torch.empty((x.shape[0], Wgu_packed.shape[1] // 2), dtype=torch.float32, device=x.device)
    mmf_glu_fwd(x, gamma, Wgu_packed, w_scales, p, stream)
    return p


def mlgru_proj(x: torch.Tensor, gamma: torch.Tensor | None, Wfcg: torch.Tensor,
               w_scales: torch.Tensor, bias: torch.Tensor | None = None,
               lb: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Returns fcg float32 [M][3d]."""
    fcg = torch.empty((x.shape[0], Wfcg.shape[1]), dtype=torch.float32, device=x.device)
    mmf_mlgru_proj(x, gamma, Wfcg, w_scales, bias, lb, fcg, None, stream)
    return fcg


def mlgru_scan(fcg: torch.Tensor, B: int, T: int, h0: torch.Tensor | None = None, stream=None):
    """Returns (o_prime float32 [B*T][d], h_last float32 [B][d])."""
    d = fcg.shape[1] // 3
    o = torch.empty((B * T, d), dtype=torch.float32, device=fcg.device)
    h = torch.empty((B, d), dtype=torch.float32, device=fcg.device)
    mmf_mlgru_scan(fcg, B, T, h0, o, h, None, stream)
    return o, h
