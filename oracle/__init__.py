"""CPU oracle for the fused BitLinear forward (arXiv 2406.02528).

TEST INFRASTRUCTURE ONLY: the test-suite, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package; the product package
``paper_2406_02528_amd`` never does, and this package never imports it.

The arithmetic lives in ``oracle.c`` (plain C, built with gcc into
``liboracle.so``); this module only marshals numpy arrays into it.  Each
wrapper names the passage of the paper it follows:

* :func:`weight_quant`   -- Algorithm 1, ``weight_quant`` (absmean ternarisation)
* :func:`pack`, :func:`unpack` -- the library's 2-bit storage format
* :func:`rms_norm`       -- the RMSNorm equation of the Loihi-methods section
  (mean of squares, eps = 1e-6, learned scale)
* :func:`act_quant`      -- Algorithm 1, ``activation_quant`` (per-token absmax)
* :func:`ternary_accumulate` -- Sec. "MatMul-free Dense Layers with Ternary
  Weights" (add where t = +1, subtract where t = -1, skip where t = 0)
* :func:`dequant`        -- Algorithm 1 (fake-quant form: integer sum times
  1/s_a times 1/s_w)
* :func:`bitlinear_fwd`  -- the composition, Algorithm 1 ``forward_pass`` with
  bias 0
* :func:`glu`, :func:`glu_fwd` -- the channel-mixer gate p = SiLU(g) (.) u of
  Sec. "MatMul-free Channel Mixer", on its own and after the two
  up-projections
* :func:`glu_interleave` -- the library's storage order for the two
  up-projection weights of one GLU (16-column blocks of gate and up in turn)
* :func:`mlgru_gates`, :func:`mlgru_scan`, :func:`add_bias`,
  :func:`mlgru_proj`, :func:`mlgru_fwd` -- the MLGRU token mixer of Sec.
  "MatMul-free Language Model Architecture": gate activations with biases
  and the forget-gate lower bound, the recurrence
  h_t = f_t h_{t-1} + (1 - f_t) c_t with the output gate o' = g sigma(h), and
  the whole mixer around its two ternary projections
* :func:`bitlinear_train_fwd`, :func:`bitlinear_bwd` -- Algorithm 1's training
  forward (the latent weights quantised on every call, rstd kept) and its
  backward_pass / rms_norm_bwd with the straight-through estimator of Sec.
  "Surrogate Gradient"
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

EPS = 1e-6  # RMSNorm epsilon stated next to the RMSNorm equation

_lib = None


def build(force: bool = True) -> str:
    """Compile ``oracle.c`` into ``liboracle.so`` with gcc (plain -O2, OpenMP,
    no fast-math, no FMA contraction)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
               "-fno-fast-math", "-ffp-contract=off", "-Wall", "-Wextra",
               _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build(force=True)
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
    lib.oracle_weight_quant.argtypes = [P, I64, I64, P, P]
    lib.oracle_weight_quant.restype = ctypes.c_int
    lib.oracle_pack.argtypes = [P, I64, I64, P]
    lib.oracle_pack.restype = ctypes.c_int
    lib.oracle_unpack.argtypes = [P, I64, I64, P]
    lib.oracle_unpack.restype = I64
    lib.oracle_rms_norm.argtypes = [P, P, I64, I64, ctypes.c_double, P, P]
    lib.oracle_act_quant.argtypes = [P, I64, I64, P, P]
    lib.oracle_ternary_accumulate.argtypes = [P, P, I64, I64, I64, P]
    lib.oracle_ternary_accumulate.restype = ctypes.c_int
    lib.oracle_ternary_accumulate_pairs.argtypes = [P, P, I64, P, P, I64, P]
    lib.oracle_ternary_accumulate_pairs.restype = ctypes.c_int
    lib.oracle_dequant.argtypes = [P, P, ctypes.c_float, I64, I64, P]
    lib.oracle_bitlinear_fwd.argtypes = [P, P, P, ctypes.c_float, I64, I64, I64,
                                         ctypes.c_double, P, P, P, P, P]
    lib.oracle_bitlinear_fwd.restype = ctypes.c_int
    lib.oracle_glu.argtypes = [P, P, I64, P]
    lib.oracle_mlgru_gates.argtypes = [P, P, P, I64, I64, P]
    lib.oracle_mlgru_scan.argtypes = [P, P, I64, I64, I64, P, P]
    lib.oracle_add_bias.argtypes = [P, P, I64, I64, P]
    lib.oracle_bitlinear_bwd.argtypes = [P, P, P, P, P, P, P, ctypes.c_float, I64, I64, I64,
                                         P, P, P, P, P, P]
    _lib = lib
    return lib


def _c(a: np.ndarray, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


def _p(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    _load().oracle_set_num_threads(int(n))


def weight_quant(W: np.ndarray):
    """Absmean ternarisation (Algorithm 1 ``weight_quant``).

    W: float32 [N][K] latent weights.  Returns (t int8 [N][K] in {-1,0,1},
    w_scale float = max(mean|W|, 1e-5), the dequantisation multiplier).
    """
    W = _c(W, np.float32)
    N, K = W.shape
    t = np.empty((N, K), np.int8)
    ws = np.zeros(1, np.float32)
    _load().oracle_weight_quant(_p(W), N, K, _p(t), _p(ws))
    return t, float(ws[0])


def pack(t: np.ndarray) -> np.ndarray:
    """Pack ternary codes t [N][K] into uint32 [K/16][N] (the library format)."""
    t = _c(t, np.int8)
    N, K = t.shape
    if K % 16:
        raise ValueError("K must be a multiple of 16")
    out = np.empty((K // 16, N), np.uint32)
    if _load().oracle_pack(_p(t), N, K, _p(out)) != 0:
        raise ValueError("codes outside {-1,0,1}")
    return out


def unpack(Wp: np.ndarray, N: int, K: int):
    """Decode uint32 [K/16][N] into t int8 [N][K].  Returns (t, n_invalid)."""
    Wp = _c(Wp, np.uint32)
    if Wp.shape != (K // 16, N) or K % 16:
        raise ValueError("bad packed shape")
    t = np.empty((N, K), np.int8)
    bad = _load().oracle_unpack(_p(Wp), N, K, _p(t))
    return t, int(bad)


def rms_norm(x: np.ndarray, gamma: np.ndarray | None, eps: float = EPS):
    """RMSNorm with the mean of squares; returns (y float32 [M][K], r float32 [M])."""
    x = _c(x, np.float32)
    M, K = x.shape
    g = None if gamma is None else _c(gamma, np.float32)
    y = np.empty((M, K), np.float32)
    r = np.empty(M, np.float32)
    _load().oracle_rms_norm(_p(x), None if g is None else _p(g), M, K,
                            float(eps), _p(y), _p(r))
    return y, r


def act_quant(y: np.ndarray):
    """Per-token absmax int8 quantisation; returns (q int8 [M][K], a_scale f32 [M])."""
    y = _c(y, np.float32)
    M, K = y.shape
    q = np.empty((M, K), np.int8)
    a = np.empty(M, np.float32)
    _load().oracle_act_quant(_p(y), M, K, _p(q), _p(a))
    return q, a


def rmsnorm_act_quant(x: np.ndarray, gamma: np.ndarray | None, eps: float = EPS):
    """RMSNorm followed by activation quantisation (the fused prologue)."""
    y, _ = rms_norm(x, gamma, eps)
    return act_quant(y)


def ternary_accumulate(q: np.ndarray, t: np.ndarray) -> np.ndarray:
    """acc int32 [M][N] = add q where t = +1, subtract where t = -1."""
    q = _c(q, np.int8)
    t = _c(t, np.int8)
    M, K = q.shape
    N, K2 = t.shape
    if K != K2:
        raise ValueError("K mismatch")
    acc = np.empty((M, N), np.int32)
    if _load().oracle_ternary_accumulate(_p(q), _p(t), M, K, N, _p(acc)) != 0:
        raise OverflowError("ternary sum outside int32 or code outside {-1,0,1}")
    return acc


def ternary_accumulate_pairs(q: np.ndarray, t: np.ndarray, ms, ns) -> np.ndarray:
    """acc for the listed (m, n) pairs only."""
    q = _c(q, np.int8)
    t = _c(t, np.int8)
    ms = _c(ms, np.int64)
    ns = _c(ns, np.int64)
    K = q.shape[1]
    out = np.empty(len(ms), np.int32)
    if _load().oracle_ternary_accumulate_pairs(_p(q), _p(t), K, _p(ms), _p(ns),
                                               len(ms), _p(out)) != 0:
        raise OverflowError("ternary sum outside int32 or code outside {-1,0,1}")
    return out


def dequant(acc: np.ndarray, a_scale: np.ndarray, w_scale: float) -> np.ndarray:
    acc = _c(acc, np.int32)
    a_scale = _c(a_scale, np.float32)
    M, N = acc.shape
    y = np.empty((M, N), np.float32)
    _load().oracle_dequant(_p(acc), _p(a_scale), ctypes.c_float(w_scale), M, N, _p(y))
    return y


def bitlinear_fwd(x: np.ndarray, gamma: np.ndarray | None, t: np.ndarray,
                  w_scale: float, eps: float = EPS):
    """Whole forward; returns dict with y, q, a_scale, acc."""
    x = _c(x, np.float32)
    t = _c(t, np.int8)
    M, K = x.shape
    N = t.shape[0]
    g = None if gamma is None else _c(gamma, np.float32)
    ybuf = np.empty((M, K), np.float32)
    q = np.empty((M, K), np.int8)
    a = np.empty(M, np.float32)
    acc = np.empty((M, N), np.int32)
    y = np.empty((M, N), np.float32)
    st = _load().oracle_bitlinear_fwd(_p(x), None if g is None else _p(g), _p(t),
                                      ctypes.c_float(w_scale), M, K, N, float(eps),
                                      _p(ybuf), _p(q), _p(a), _p(acc), _p(y))
    if st != 0:
        raise OverflowError("ternary sum outside int32")
    return {"y": y, "q": q, "a_scale": a, "acc": acc}


def glu(g: np.ndarray, u: np.ndarray) -> np.ndarray:
    """p = SiLU(g) * u elementwise (fp64, rounded to fp32 once)."""
    g = _c(g, np.float32)
    u = _c(u, np.float32)
    if g.shape != u.shape:
        raise ValueError("g and u differ in shape")
    p = np.empty(g.shape, np.float32)
    _load().oracle_glu(_p(g), _p(u), g.size, _p(p))
    return p


def glu_fwd(x: np.ndarray, gamma: np.ndarray | None, t_g: np.ndarray, w_scale_g: float,
            t_u: np.ndarray, w_scale_u: float, eps: float = EPS):
    """The channel mixer's up-projections and gate: g = BitLinear(x; t_g),
    u = BitLinear(x; t_u), both after the same RMSNorm and activation
    quantisation, then p = SiLU(g) * u.  Returns dict with p, g, u, acc_g, acc_u."""
    og = bitlinear_fwd(x, gamma, t_g, w_scale_g, eps)
    ou = bitlinear_fwd(x, gamma, t_u, w_scale_u, eps)
    return {"p": glu(og["y"], ou["y"]), "g": og["y"], "u": ou["y"],
            "acc_g": og["acc"], "acc_u": ou["acc"], "q": og["q"], "a_scale": og["a_scale"]}


def glu_interleave(t_g: np.ndarray, t_u: np.ndarray) -> np.ndarray:
    """Rows of the combined [2L][K] code matrix in the library's GLU order:
    blocks of 16 gate rows and 16 up rows in turn (rows 32b .. 32b+15 are gate
    rows 16b .. 16b+15, rows 32b+16 .. 32b+31 the up rows with the same
    indices).  L must be a multiple of 16."""
    t_g = np.asarray(t_g)
    t_u = np.asarray(t_u)
    L, K = t_g.shape
    if t_u.shape != (L, K) or L % 16:
        raise ValueError("gate and up must both be [L][K] with L a multiple of 16")
    out = np.empty((2 * L, K), t_g.dtype)
    for b in range(L // 16):
        out[32 * b:32 * b + 16] = t_g[16 * b:16 * b + 16]
        out[32 * b + 16:32 * b + 32] = t_u[16 * b:16 * b + 16]
    return out


def _opt(a, dtype):
    return None if a is None else _c(a, dtype)


def mlgru_gates(z: np.ndarray, bias: np.ndarray | None = None,
                lb: np.ndarray | None = None) -> np.ndarray:
    """Gate activations of the MLGRU.  z is [M][3d] (forget | candidate |
    output-gate projections); returns fcg [M][3d] with f = lb + (1 - lb)
    sigma(z_f + b_f), c = SiLU(z_c + b_c), g = z_g + b_g (fp64, rounded once)."""
    z = _c(z, np.float32)
    M, n3 = z.shape
    if n3 % 3:
        raise ValueError("z must have 3d columns")
    d = n3 // 3
    b = _opt(bias, np.float32)
    low = _opt(lb, np.float32)
    if b is not None and b.shape != (3 * d,):
        raise ValueError("bias must be [3d]")
    if low is not None and low.shape != (d,):
        raise ValueError("lb must be [d]")
    out = np.empty((M, 3 * d), np.float32)
    _load().oracle_mlgru_gates(_p(z), None if b is None else _p(b),
                               None if low is None else _p(low), M, d, _p(out))
    return out


def mlgru_scan(fcg: np.ndarray, B: int, T: int, h0: np.ndarray | None = None):
    """The MLGRU recurrence and output gate over B sequences of T tokens
    (rows b*T + t of fcg [B*T][3d]).  Returns (o' [B*T][d], h_last [B][d])."""
    fcg = _c(fcg, np.float32)
    if fcg.shape[0] != B * T or fcg.shape[1] % 3:
        raise ValueError("fcg must be [B*T][3d]")
    d = fcg.shape[1] // 3
    h = _opt(h0, np.float32)
    if h is not None and h.shape != (B, d):
        raise ValueError("h0 must be [B][d]")
    o = np.empty((B * T, d), np.float32)
    hl = np.empty((B, d), np.float32)
    _load().oracle_mlgru_scan(_p(fcg), None if h is None else _p(h), B, T, d, _p(o), _p(hl))
    return o, hl


def add_bias(y: np.ndarray, b: np.ndarray) -> np.ndarray:
    """y + b per row (fp64, rounded once): the bias of Algorithm 1's forward."""
    y = _c(y, np.float32)
    b = _c(b, np.float32)
    M, N = y.shape
    if b.shape != (N,):
        raise ValueError("bias must be [N]")
    out = np.empty((M, N), np.float32)
    _load().oracle_add_bias(_p(y), _p(b), M, N, _p(out))
    return out


def mlgru_proj(x: np.ndarray, gamma: np.ndarray | None, t_fcg: np.ndarray, w_scales,
               bias: np.ndarray | None = None, lb: np.ndarray | None = None, eps: float = EPS):
    """The MLGRU's input projections and gate activations: the three ternary
    projections of the normalised, quantised x (one RMSNorm, one activation
    quantisation; t_fcg [3d][K] holds W_f, W_c, W_g in turn, segment s scaled
    by w_scales[s]), then :func:`mlgru_gates`.  Returns dict with fcg, z, acc,
    q, a_scale."""
    t_fcg = _c(t_fcg, np.int8)
    d = t_fcg.shape[0] // 3
    if t_fcg.shape[0] != 3 * d:
        raise ValueError("t_fcg must have 3d rows")
    parts = [bitlinear_fwd(x, gamma, t_fcg[s * d:(s + 1) * d], float(w_scales[s]), eps)
             for s in range(3)]
    z = np.concatenate([p["y"] for p in parts], axis=1)
    acc = np.concatenate([p["acc"] for p in parts], axis=1)
    return {"fcg": mlgru_gates(z, bias, lb), "z": z, "acc": acc,
            "q": parts[0]["q"], "a_scale": parts[0]["a_scale"]}


def mlgru_fwd(x: np.ndarray, B: int, T: int, gamma: np.ndarray | None, t_fcg: np.ndarray,
              w_scales, bias: np.ndarray | None, lb: np.ndarray | None,
              h0: np.ndarray | None, gamma_o: np.ndarray | None, t_o: np.ndarray,
              w_scale_o: float, b_o: np.ndarray | None, eps: float = EPS):
    """The whole MLGRU token mixer over B sequences of T tokens (x rows
    b*T + t): projections and gates, recurrence and output gate, then the
    output projection o = BitLinear(o'; t_o) + b_o.  Returns dict with o,
    h_last, o_prime, fcg and the output projection's q, acc, a_scale."""
    pr = mlgru_proj(x, gamma, t_fcg, w_scales, bias, lb, eps)
    o_prime, h_last = mlgru_scan(pr["fcg"], B, T, h0)
    out = bitlinear_fwd(o_prime, gamma_o, t_o, w_scale_o, eps)
    o = out["y"] if b_o is None else add_bias(out["y"], b_o)
    return {"o": o, "h_last": h_last, "o_prime": o_prime, "fcg": pr["fcg"],
            "y_o": out["y"], "q_o": out["q"], "acc_o": out["acc"], "a_scale_o": out["a_scale"]}


def bitlinear_train_fwd(x: np.ndarray, gamma: np.ndarray | None, W: np.ndarray,
                        bias: np.ndarray | None = None, eps: float = EPS):
    """Algorithm 1's forward_pass with the latent weights W [N][K]:
    weight_quant, RMSNorm (rstd kept for the backward), activation_quant,
    the ternary product, the bias.  Returns dict with y, t, w_scale, q,
    a_scale, rstd, acc."""
    t, ws = weight_quant(W)
    out = bitlinear_fwd(x, gamma, t, ws, eps)
    _, r = rms_norm(x, gamma, eps)
    y = out["y"] if bias is None else add_bias(out["y"], bias)
    return {"y": y, "t": t, "w_scale": ws, "q": out["q"], "a_scale": out["a_scale"],
            "rstd": r, "acc": out["acc"]}


def bitlinear_bwd(dO: np.ndarray, x: np.ndarray, gamma: np.ndarray | None, rstd: np.ndarray,
                  q: np.ndarray, a_scale: np.ndarray, t: np.ndarray, w_scale: float):
    """Backward of the BitLinear (Algorithm 1 backward_pass, rms_norm_bwd in the
    RMSNorm reading, straight-through quantisers).  dO [M][N] (values of the
    bf16 gradient), x [M][K], rstd [M] the forward's, q/a_scale the forward's
    int8 activations, t [N][K] the forward's ternary codes.  Returns dict with
    dx [M][K], dW [N][K], db [N], dgamma [K] (at gamma = 1 without gamma),
    dY [M][K] (fp64), yq [M][K] (the bf16-stored dequantised activations)."""
    dO = _c(dO, np.float32)
    x = _c(x, np.float32)
    M, K = x.shape
    N = dO.shape[1]
    g = None if gamma is None else _c(gamma, np.float32)
    r = _c(rstd, np.float32)
    q = _c(q, np.int8)
    a = _c(a_scale, np.float32)
    t = _c(t, np.int8)
    if dO.shape != (M, N) or t.shape != (N, K) or q.shape != (M, K):
        raise ValueError("shape mismatch")
    dY = np.empty((M, K), np.float64)
    yq = np.empty((M, K), np.float32)
    dx = np.empty((M, K), np.float32)
    dW = np.empty((N, K), np.float32)
    db = np.empty(N, np.float32)
    dg = np.empty(K, np.float32)
    _load().oracle_bitlinear_bwd(_p(dO), _p(x), None if g is None else _p(g), _p(r), _p(q), _p(a),
                                 _p(t), ctypes.c_float(w_scale), M, K, N, _p(dY), _p(yq), _p(dx),
                                 _p(dW), _p(db), _p(dg))
    return {"dx": dx, "dW": dW, "db": db, "dgamma": dg, "dY": dY, "yq": yq}
