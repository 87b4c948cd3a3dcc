"""GPU parity of the MLGRU token mixer (Sec. "MatMul-free Language Model
Architecture", paragraph "MatMul-free Linear Gated Recurrent Unit" and its
equations) through the C ABI, against the CPU oracle on the same seeded
inputs.  Each stage is checked on the previous stage's GPU output, and the
whole-mixer entry point must equal the three stage calls bit for bit.

Bars, with u = 2^-24 the fp32 unit roundoff:
  * packed f|c|g words: bit-exact; q: the activation-quantisation bar (at most
    1 LSB apart in at most 0.1% of entries);
  * gates, on rows whose q match: the library forms y = fp32(acc) *
    fp32(a_scale w_scale) (two roundings, the oracle's one: 3u|y|, plus the
    relative difference r_a of the two sides' a_scale, measured per row), then
    z = y + b (rounded on both sides: 2u|z|) and the activation in fp32 (the
    hardware exp2 and reciprocal, 1 ulp each, the argument -z log2 e rounded
    once: the sigmoid s is within (1 - s)(|z| + 2) u + 3u relative, its |z|
    part at most u / 4 absolute for f and at most u z^2 s (1 - s) < u / 2 for
    c; within 8u of the result in all).  With e_z = (3u + r_a)|y| + 2u|z|:
      |df| <= (1 - lb) e_z / 4 + 8u     (the sigmoid's slope is at most 1/4)
      |dc| <= 1.1 e_z + 8u |c|           (SiLU's slope lies in (-0.1, 1.1))
      |dg| <= e_z
    on rows with a flip in q the pre-activation may move by 1e-3 of the row's
    largest |z| in that segment, scaled by the same slopes;
  * dense layer with bias: |dy| <= (3u + r_a) |y| + 2u |y + b| per element, the
    row bound 1e-3 max|y| on rows with a flip in q;
  * recurrence, on the same gates: with m_t = f_t m_{t-1} + (1 - f_t)|c_t|
    (m_0 = |h_0|, a bound on |h_t|) and S_t = f_t S_{t-1} + m_t, the fp32
    recurrence taken token by token stays within 4u S_t of the exact state
    (each step rounds terms bounded by m_t, and errors decay as the state
    does).  The library composes chunks of L tokens (and runs of chunks) into
    maps h -> A h + B: a product of P forget gates carries relative error
    (P - 1)u, and P (prod f) |h| <= S_t, so each level of composition and each
    join adds at most a few u S_t, as does the second pass over each chunk.  The output gate's sigmoid s comes from the
    hardware exp2 and reciprocal with the argument -h log2 e rounded once:
    relative error (1 - s)(|h| + 2) u + 3u, whose |h| part is at most
    s (1 - s) |h| u <= u / 4 in absolute terms.  So the test allows
      |dh_t| <= 2 (L + 8) u S_t,   |do'_t| <= |g_t| (|dh_t| + u) / 4 + 6u |o'_t|.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from _parity import compare_q, dev, log, packed_to_np, to_dev_x

pytestmark = pytest.mark.gpu

U = 2.0 ** -24
ROW_REL = 1e-3


@pytest.fixture(scope="module")
def mmf():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2406_02528_amd as m
    return m


def T_(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev())


def opt(a):
    return None if a is None else T_(a)


def chunk_len(T: int) -> int:
    # chunk length of the library's recurrence (at most 128 chunks, at least 16 tokens)
    return T if T <= 16 else max(16, -(-T // 128))


# --------------------------------------------------------------------------
# bars
# --------------------------------------------------------------------------

def a_rel(a_gpu: np.ndarray, a_ref: np.ndarray) -> np.ndarray:
    """Per-row relative difference of the two sides' a_scale."""
    a = a_ref.astype(np.float64)
    return np.abs(a_gpu.astype(np.float64) - a) / a


def check_gates(fcg_gpu, z_ref, bias, lb, flip_mask, ra):
    """fcg_gpu [M][3d] against the oracle's pre-activations z_ref (no bias);
    ra: per-row relative a_scale difference."""
    M, n3 = z_ref.shape
    d = n3 // 3
    y = z_ref.astype(np.float64)
    b = np.zeros(n3) if bias is None else bias.astype(np.float64)
    z = y + b
    ref = oracle.mlgru_gates(z_ref, bias, lb).astype(np.float64)
    got = fcg_gpu.astype(np.float64)
    low = np.zeros(d) if lb is None else lb.astype(np.float64)
    e_z = (3 * U + ra[:, None]) * np.abs(y) + 2 * U * np.abs(z)
    # rows with a flipped q: the pre-activation may move by 1e-3 of the
    # segment's largest |z|
    for s in range(3):
        seg = np.s_[s * d:(s + 1) * d]
        shift = ROW_REL * np.abs(z[:, seg]).max(axis=1, keepdims=True) * flip_mask[:, None]
        e_z[:, seg] += shift
    err = np.abs(got - ref)
    bounds = [(1 - low) * e_z[:, :d] / 4 + 8 * U,
              1.1 * e_z[:, d:2 * d] + 8 * U * np.abs(ref[:, d:2 * d]) + 1e-30,
              e_z[:, 2 * d:] + 1e-30]
    for s, name in enumerate("fcg"):
        seg = np.s_[s * d:(s + 1) * d]
        bad = ~(err[:, seg] <= bounds[s])   # NaN counts as out of bound
        if bad.any():
            m, n = np.argwhere(bad)[0]
            n += s * d
            raise AssertionError(
                f"{name}: {int(bad.sum())} values out of bound, worst excess "
                f"{float((err[:, seg] - bounds[s]).max()):.3e}; first at ({m},{n}): y={y[m, n]!r} "
                f"z={z[m, n]!r} got={got[m, n]!r} ref={ref[m, n]!r} r_a={ra[m]:.3e}")
    return float((err / (np.abs(ref) + 1e-30)).max(initial=0.0))


def scan_bounds(fcg, B, T, h0):
    """Per-token bounds on the state error (|dh_t|) of the library's chunked
    fp32 recurrence, [B*T][d]."""
    d = fcg.shape[1] // 3
    f = fcg[:, :d].astype(np.float64).reshape(B, T, d)
    ac = np.abs(fcg[:, d:2 * d].astype(np.float64)).reshape(B, T, d)
    m = np.zeros((B, d)) if h0 is None else np.abs(h0.astype(np.float64))
    S = np.zeros((B, d))
    L = chunk_len(T)
    out = np.empty((B, T, d))
    for t in range(T):
        m = f[:, t] * m + (1 - f[:, t]) * ac[:, t]
        S = f[:, t] * S + m
        out[:, t] = 2 * (L + 8) * U * S
    return out.reshape(B * T, d)


def check_scan(o_gpu, h_gpu, fcg, B, T, h0):
    d = fcg.shape[1] // 3
    o_ref, h_ref = oracle.mlgru_scan(fcg, B, T, h0)
    tol_h = scan_bounds(fcg, B, T, h0)
    g = np.abs(fcg[:, 2 * d:].astype(np.float64))
    tol_o = g * (tol_h + U) / 4 + 6 * U * np.abs(o_ref.astype(np.float64)) + 1e-30
    err_o = np.abs(o_gpu.astype(np.float64) - o_ref)
    bad = ~(err_o <= tol_o)
    assert not bad.any(), f"o': {int(bad.sum())} out of bound, worst excess {float((err_o - tol_o).max()):.3e}"
    if h_gpu is not None:
        last = tol_h.reshape(B, T, d)[:, -1]
        err_h = np.abs(h_gpu.astype(np.float64) - h_ref)
        assert not (err_h > last + 1e-30).any(), f"h_last worst excess {float((err_h - last).max()):.3e}"
    return float((err_o / (np.abs(o_ref) + 1e-30)).max(initial=0.0))


def check_bias_out(y_gpu, y_ref, b, flip_mask, ra):
    y = y_ref.astype(np.float64)
    out = oracle.add_bias(y_ref, b).astype(np.float64)
    tol = (3 * U + ra[:, None]) * np.abs(y) + 2 * U * np.abs(out) + 1e-30
    tol = tol + ROW_REL * np.abs(y).max(axis=1, keepdims=True) * flip_mask[:, None]
    err = np.abs(y_gpu.astype(np.float64) - out)
    bad = ~(err <= tol)   # NaN counts as out of bound
    assert not bad.any(), f"{int(bad.sum())} outputs out of bound, worst excess {float((err - tol).max()):.3e}"


def flips(q_gpu: np.ndarray, q_ref: np.ndarray) -> np.ndarray:
    rows, _ = compare_q(q_gpu, q_ref)
    mask = np.zeros(q_ref.shape[0], bool)
    mask[rows] = True
    return mask


def quantise_gpu(mmf, x_d, g_d, M, K):
    """The library's int8 activations and a_scale of x (bf16 or float32)."""
    q = torch.empty((M, K), dtype=torch.int8, device=dev())
    a = torch.empty((M,), dtype=torch.float32, device=dev())
    mmf.mmf_act_quant(x_d, g_d, q, a)
    torch.cuda.synchronize()
    return q.cpu().numpy(), a.cpu().numpy()


def pack_fcg(mmf, W, joint: bool):
    """Ternarise the stacked [3d][K] latent weights jointly (one scale) or per
    gate; returns (Wfcg [K/16][3d], w_scales [3] tensor, t [3d][K], scales)."""
    d = W.shape[0] // 3
    if joint:
        t, ws = oracle.weight_quant(W)
        Wp, wsd = mmf.ternarize(T_(W))
        scales = [ws] * 3
        w_scales = torch.cat([wsd, wsd, wsd])
    else:
        parts = [oracle.weight_quant(W[s * d:(s + 1) * d]) for s in range(3)]
        t = np.concatenate([p[0] for p in parts])
        scales = [p[1] for p in parts]
        packs = [mmf.ternarize(T_(W[s * d:(s + 1) * d])) for s in range(3)]
        Wp = torch.cat([p[0] for p in packs], dim=1).contiguous()
        w_scales = torch.cat([p[1] for p in packs])
    torch.cuda.synchronize()
    assert np.array_equal(packed_to_np(Wp), oracle.pack(t)), "packed f|c|g words differ"
    assert w_scales.cpu().numpy().tolist() == [np.float32(s) for s in scales]
    return Wp, w_scales, t, scales


# --------------------------------------------------------------------------
# input projections and gates
# --------------------------------------------------------------------------

@pytest.mark.parametrize("M,path", [(1, 0), (8, 0), (17, 0), (17, 1), (300, 0)])
def test_mlgru_proj_random_shapes(mmf, M, path):
    rs = np.random.default_rng(3000 + M + 7 * path)
    prev = mmf.mmf_set_path(path)
    try:
        for K in (16, 64, 2064):
            for d in (16, 48, 160):
                joint = bool((K + d) % 2)
                bits, xf, gamma, W = workloads.random_case(rs, M, K, 3 * d)
                bias = rs.uniform(-0.5, 0.5, 3 * d).astype(np.float32) if d != 48 else None
                lb = rs.uniform(0.0, 0.95, d).astype(np.float32) if K != 64 else None
                log(f"[mlgru proj] M={M} K={K} d={d} path={path} joint={joint} "
                    f"bias={bias is not None} lb={lb is not None}")
                Wp, w_scales, t, scales = pack_fcg(mmf, W, joint)
                ref = oracle.mlgru_proj(xf, gamma, t, scales, bias, lb)
                x_d, g_d = to_dev_x(bits), T_(gamma)
                fcg = torch.full((M, 3 * d), float("nan"), dtype=torch.float32, device=dev())
                mmf.mmf_mlgru_proj(x_d, g_d, Wp, w_scales, opt(bias), opt(lb), fcg)
                q, a = quantise_gpu(mmf, x_d, g_d, M, K)
                check_gates(fcg.cpu().numpy(), ref["z"], bias, lb, flips(q, ref["q"]),
                            a_rel(a, ref["a_scale"]))
    finally:
        mmf.mmf_set_path(prev)


def test_mlgru_proj_contraction_stage_matches(mmf):
    # from quantised activations the MFMA kernel gives the projection's bits
    rs = np.random.default_rng(3100)
    M, K, d = 70, 256, 48
    bits, xf, gamma, W = workloads.random_case(rs, M, K, 3 * d)
    Wp, w_scales, _, _ = pack_fcg(mmf, W, False)
    bias, lb = T_(rs.uniform(-0.5, 0.5, 3 * d).astype(np.float32)), T_(rs.uniform(0, 0.9, d).astype(np.float32))
    x_d, g_d = to_dev_x(bits), T_(gamma)
    f1 = mmf.mlgru_proj(x_d, g_d, Wp, w_scales, bias, lb)
    q = torch.empty((M, K), dtype=torch.int8, device=dev())
    a = torch.empty((M,), dtype=torch.float32, device=dev())
    r = torch.empty((M,), dtype=torch.int32, device=dev())
    mmf.mmf_act_quant(x_d, g_d, q, a, r)
    f2 = torch.empty_like(f1)
    mmf.mmf_mlgru_proj_q(q, a, r, Wp, w_scales, bias, lb, f2)
    torch.cuda.synchronize()
    assert torch.equal(f1, f2)


@pytest.mark.parametrize("M", [1, 5, 300])
def test_bitlinear_bias(mmf, M):
    rs = np.random.default_rng(4000 + M)
    for K, N in ((64, 36), (2048, 2048)):
        bits, xf, gamma, W = workloads.random_case(rs, M, K, N)
        b = rs.uniform(-0.5, 0.5, N).astype(np.float32)
        log(f"[bias] M={M} K={K} N={N}")
        t, ws = oracle.weight_quant(W)
        Wp, wsd = mmf.ternarize(T_(W))
        ref = oracle.bitlinear_fwd(xf, gamma, t, ws)
        x_d, g_d = to_dev_x(bits), T_(gamma)
        y = torch.full((M, N), float("nan"), dtype=torch.float32, device=dev())
        mmf.mmf_bitlinear_fwd_bias(x_d, g_d, Wp, wsd, T_(b), y)
        # float32 input (the mixer's o' form)
        y32 = torch.full((M, N), float("nan"), dtype=torch.float32, device=dev())
        mmf.mmf_bitlinear_fwd_bias(T_(xf), g_d, Wp, wsd, T_(b), y32)
        q, a = quantise_gpu(mmf, x_d, g_d, M, K)
        fm, ra = flips(q, ref["q"]), a_rel(a, ref["a_scale"])
        check_bias_out(y.cpu().numpy(), ref["y"], b, fm, ra)
        check_bias_out(y32.cpu().numpy(), ref["y"], b, fm, ra)
        # with a zero bias the result is the plain forward's, bit for bit
        y0 = torch.empty_like(y)
        mmf.mmf_bitlinear_fwd_bias(x_d, g_d, Wp, wsd, torch.zeros(N, device=dev()), y0)
        yp = mmf.bitlinear(x_d, g_d, Wp, wsd)
        torch.cuda.synchronize()
        assert torch.equal(y0, yp)


# --------------------------------------------------------------------------
# recurrence
# --------------------------------------------------------------------------

SCAN_CASES = [
    # B, T, d, initial state, in place, store h_last
    (1, 1, 16, True, True, True),
    (3, 1, 48, False, False, True),
    (2, 16, 32, True, False, True),
    (2, 17, 32, True, False, True),
    (1, 33, 16, False, True, True),
    (1, 300, 64, True, True, True),
    (4, 1000, 160, True, False, False),
    (2, 5000, 16, False, False, True),
]


@pytest.mark.parametrize("B,T,d,with_h0,inplace,store", SCAN_CASES)
def test_mlgru_scan(mmf, B, T, d, with_h0, inplace, store):
    rs = np.random.default_rng(5000 + B * 7 + T + d)
    fcg = workloads.random_gates(rs, B * T, d)
    h0 = rs.standard_normal((B, d)).astype(np.float32) if with_h0 else None
    log(f"[mlgru scan] B={B} T={T} d={d} h0={with_h0} inplace={inplace} store={store}")
    o = torch.full((B * T, d), float("nan"), dtype=torch.float32, device=dev())
    h0_d = opt(h0)
    if inplace and h0_d is not None:
        h_d = h0_d
    else:
        h_d = torch.full((B, d), float("nan"), dtype=torch.float32, device=dev()) if store else None
    mmf.mmf_mlgru_scan(T_(fcg), B, T, h0_d, o, h_d)
    torch.cuda.synchronize()
    worst = check_scan(o.cpu().numpy(), None if h_d is None else h_d.cpu().numpy(), fcg, B, T, h0)
    log(f"  worst rel o' {worst:.2e}")
    # caller workspace gives the same bits
    need = mmf.mmf_mlgru_scan_workspace_bytes(B, T, d)
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev())
    o2 = torch.empty_like(o)
    mmf.mmf_mlgru_scan(T_(fcg), B, T, opt(h0), o2, None, ws if need else None)
    torch.cuda.synchronize()
    assert torch.equal(o, o2)


def test_mlgru_scan_no_state_is_zero_state(mmf):
    rs = np.random.default_rng(61)
    B, T, d = 2, 100, 32
    fcg = T_(workloads.random_gates(rs, B * T, d))
    o1, h1 = mmf.mlgru_scan(fcg, B, T, None)
    o2, h2 = mmf.mlgru_scan(fcg, B, T, torch.zeros((B, d), device=dev()))
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(h1, h2)


def test_mlgru_decode_steps_continue_the_sequence(mmf):
    # T single-token calls, the state carried in place, against one call
    # over the whole sequence (the same recurrence, one token per chunk)
    rs = np.random.default_rng(62)
    B, T, d = 3, 24, 48
    fcg = workloads.random_gates(rs, B * T, d)
    h0 = rs.standard_normal((B, d)).astype(np.float32)
    h = T_(h0)
    steps = []
    rows = fcg.reshape(B, T, 3 * d)
    for t in range(T):
        o = torch.empty((B, d), dtype=torch.float32, device=dev())
        mmf.mmf_mlgru_scan(T_(rows[:, t]), B, 1, h, o, h)
        steps.append(o)
    torch.cuda.synchronize()
    o_steps = torch.stack(steps, dim=1).reshape(B * T, d).cpu().numpy()
    check_scan(o_steps, h.cpu().numpy(), fcg, B, T, h0)


# --------------------------------------------------------------------------
# the whole mixer
# --------------------------------------------------------------------------

def run_mixer(mmf, inp, B, T, with_state=True):
    """Whole-mixer call and the three stage calls on device copies of inp;
    returns dict of numpy results of both, and the stage intermediates."""
    d = inp["W_o"].shape[0]
    Wp, w_scales, t, scales = pack_fcg(mmf, inp["W_fcg"], True)
    Wo, wso = mmf.ternarize(T_(inp["W_o"]))
    x_d, g_d, go_d = to_dev_x(inp["x_bits"]), T_(inp["gamma"]), T_(inp["gamma_o"])
    bias, lb, b_o = T_(inp["bias"]), T_(inp["lb"]), T_(inp["b_o"])
    h0 = T_(inp["h0"]) if with_state else None
    M = B * T
    o = torch.full((M, d), float("nan"), dtype=torch.float32, device=dev())
    h_last = torch.full((B, d), float("nan"), dtype=torch.float32, device=dev())
    mmf.mmf_mlgru_fwd(x_d, B, T, g_d, Wp, w_scales, bias, lb, h0, h_last, go_d, Wo, wso, b_o, o)
    # stages
    fcg = mmf.mlgru_proj(x_d, g_d, Wp, w_scales, bias, lb)
    op, h_s = mmf.mlgru_scan(fcg, B, T, h0)
    o_s = torch.empty_like(o)
    mmf.mmf_bitlinear_fwd_bias(op, go_d, Wo, wso, b_o, o_s)
    q_in, a_in = quantise_gpu(mmf, x_d, g_d, M, d)
    q_o, a_o = quantise_gpu(mmf, op, go_d, M, d)
    torch.cuda.synchronize()
    assert torch.equal(o, o_s), "whole mixer differs from its stages"
    assert torch.equal(h_last, h_s)
    t_o, ws_o = oracle.weight_quant(inp["W_o"])
    return {"o": o.cpu().numpy(), "h_last": h_last.cpu().numpy(), "fcg": fcg.cpu().numpy(),
            "op": op.cpu().numpy(), "q_in": q_in, "q_o": q_o, "a_in": a_in, "a_o": a_o,
            "t": t, "scales": scales,
            "t_o": t_o, "ws_o": ws_o}


@pytest.mark.parametrize("B,T,d", [(1, 1, 64), (3, 1, 48), (2, 40, 32), (1, 300, 128)])
def test_mlgru_fwd_random(mmf, B, T, d):
    rs = np.random.default_rng(7000 + B + T + d)
    bits, xf, gamma, W = workloads.random_case(rs, B * T, d, 3 * d)
    inp = {"x_bits": bits, "x_f32": xf, "gamma": gamma, "W_fcg": W,
           "W_o": (rs.standard_normal((d, d)) * 0.02).astype(np.float32),
           "gamma_o": rs.uniform(0.5, 1.5, d).astype(np.float32),
           "bias": rs.uniform(-0.5, 0.5, 3 * d).astype(np.float32),
           "b_o": rs.uniform(-0.5, 0.5, d).astype(np.float32),
           "lb": rs.uniform(0.0, 0.95, d).astype(np.float32),
           "h0": rs.standard_normal((B, d)).astype(np.float32)}
    log(f"[mlgru fwd] B={B} T={T} d={d}")
    r = run_mixer(mmf, inp, B, T)
    # stage by stage against the oracle, each on the GPU's previous output
    pr = oracle.mlgru_proj(xf, gamma, r["t"], r["scales"], inp["bias"], inp["lb"])
    check_gates(r["fcg"], pr["z"], inp["bias"], inp["lb"], flips(r["q_in"], pr["q"]),
                a_rel(r["a_in"], pr["a_scale"]))
    check_scan(r["op"], r["h_last"], r["fcg"], B, T, inp["h0"])
    out = oracle.bitlinear_fwd(r["op"], inp["gamma_o"], r["t_o"], r["ws_o"])
    check_bias_out(r["o"], out["y"], inp["b_o"], flips(r["q_o"], out["q"]),
                   a_rel(r["a_o"], out["a_scale"]))


@pytest.mark.parametrize("name", ["mlgru_decode", "mlgru_prefill"])
def test_mlgru_workloads(mmf, name):
    """The decode step (B=1, T=1) and the 2048-token prefill at d = 2048:
    whole rows of every stage for the decode step; for the prefill the whole
    recurrence and sampled projection outputs (256 rows)."""
    w = workloads.MLGRU_WORKLOADS[name]
    inp = workloads.make_mlgru(w)
    log(f"[{name}] B={w.B} T={w.T} d={w.d}")
    r = run_mixer(mmf, inp, w.B, w.T)
    rows = np.arange(w.M) if w.M <= 8 else np.unique(np.concatenate(
        [np.random.default_rng(8).integers(0, w.M, 252), [0, 1, w.M - 2, w.M - 1]]))
    pr = oracle.mlgru_proj(inp["x_f32"][rows], inp["gamma"], r["t"], r["scales"], inp["bias"], inp["lb"])
    check_gates(r["fcg"][rows], pr["z"], inp["bias"], inp["lb"], flips(r["q_in"][rows], pr["q"]),
                a_rel(r["a_in"][rows], pr["a_scale"]))
    log(f"[{name}] recurrence")
    check_scan(r["op"], r["h_last"], r["fcg"], w.B, w.T, inp["h0"])
    out = oracle.bitlinear_fwd(r["op"][rows], inp["gamma_o"], r["t_o"], r["ws_o"])
    check_bias_out(r["o"][rows], out["y"], inp["b_o"], flips(r["q_o"][rows], out["q"]),
                   a_rel(r["a_o"][rows], out["a_scale"]))


@pytest.mark.parametrize("B,d", [(1, 2048), (5, 96), (21, 64)])
def test_mlgru_decode_step_fused_equals_in_place(mmf, B, d):
    """A decode step (T = 1) whose new state goes to its own array runs the
    recurrence and output gate in the output projection's prologue; with the
    state updated in place it runs the recurrence kernel and the plain
    projection.  Same arithmetic: the same bits (B = 21 spans two 16-token
    slices)."""
    rs = np.random.default_rng(7700 + B + d)
    bits, xf, gamma, W = workloads.random_case(rs, B, d, 3 * d)
    Wp, w_scales, _, _ = pack_fcg(mmf, W, True)
    Wo, wso = mmf.ternarize(T_((rs.standard_normal((d, d)) * 0.02).astype(np.float32)))
    x_d, g_d = to_dev_x(bits), T_(gamma)
    go = T_(rs.uniform(0.5, 1.5, d).astype(np.float32))
    bias = T_(rs.uniform(-0.5, 0.5, 3 * d).astype(np.float32))
    lb = T_(rs.uniform(0.0, 0.95, d).astype(np.float32))
    b_o = T_(rs.uniform(-0.5, 0.5, d).astype(np.float32))
    h0 = rs.standard_normal((B, d)).astype(np.float32)
    log(f"[mlgru step] B={B} d={d}")
    o1 = torch.empty((B, d), dtype=torch.float32, device=dev())
    h_in, h_out = T_(h0), torch.full((B, d), float("nan"), dtype=torch.float32, device=dev())
    mmf.mmf_mlgru_fwd(x_d, B, 1, g_d, Wp, w_scales, bias, lb, h_in, h_out, go, Wo, wso, b_o, o1)
    o2 = torch.empty_like(o1)
    h_ip = T_(h0)
    mmf.mmf_mlgru_fwd(x_d, B, 1, g_d, Wp, w_scales, bias, lb, h_ip, h_ip, go, Wo, wso, b_o, o2)
    o3 = torch.empty_like(o1)   # no state at all: h_0 = 0, nothing stored
    mmf.mmf_mlgru_fwd(x_d, B, 1, g_d, Wp, w_scales, bias, lb, None, None, go, Wo, wso, b_o, o3)
    o4 = torch.empty_like(o1)
    h_zero = torch.zeros((B, d), dtype=torch.float32, device=dev())
    mmf.mmf_mlgru_fwd(x_d, B, 1, g_d, Wp, w_scales, bias, lb, h_zero, h_zero, go, Wo, wso, b_o, o4)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(h_out, h_ip)
    assert torch.equal(o3, o4)
    assert torch.equal(h_in, T_(h0))   # the fused path leaves the input state alone
