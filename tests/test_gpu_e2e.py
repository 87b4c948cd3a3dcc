"""End-to-end GPU parity of the widened paths, from the inputs alone.

The staged tests (test_gpu_mlgru.py, test_gpu_train.py) check each stage on
the previous stage's GPU output.  Here the oracle runs the whole chain from x
(with the latent weights and, for the backward, the output gradient) and the
library runs its whole entry points on the same inputs; the final results are
compared with a bound propagated through the stages from the oracle's own
intermediate values.  No GPU result enters an expected value; the only GPU
intermediates the tests read are the quantised input activations, a_scale and
rstd, each held to its own bar first (q: at most 1 LSB apart in at most 0.1%
of entries; a_scale within 8u relative; rstd within one ulp), and the rows
where q differs then take the row allowance.

MLGRU token mixer (Sec. "MatMul-free Language Model Architecture", paragraph
"MatMul-free Linear Gated Recurrent Unit" and its equations), u = 2^-24:
  1. gates: the projection bar of test_gpu_mlgru.py with r_a = 8u, giving
     bounds Bf, Bc, Bg on the forget gate, candidate and output gate;
  2. recurrence: the gate errors carried through the exact recurrence,
       D_t = f D_{t-1} + Bf (|h_{t-1}| + D_{t-1} + |c| + Bc) + (1 - f + Bf) Bc
     (D_0 = 0), plus the library's rounding bound 2 (L + 8) u S_t of its
     chunked fp32 recurrence (S_t over the perturbed gates), e_t in all; for
     the gated output o' = g s(h):
       |do'| <= Bg (s(h) + (e + u) / 4) + |g| (e + u) / 4 + 6u (|o'| + Bg);
     h_last within e_T;
  3. output projection on o': the row's a_scale moves by at most the largest
     perturbation of |o' gamma| over its maximum, plus the movement of rstd
     (sum |o'| do' / (sum o'^2 + K eps)), plus 8u: r_a; q can differ from
     the oracle's only where 127 o' gamma / max|o' gamma| lies within its own
     movement of a rounding midpoint, and rows with such an element get the
     1e-3 row allowance; every element gets (3u + r_a)|y| + 2u|o|.

Training step (Algorithm 1 forward_pass with the latent weights, then
backward_pass and rms_norm_bwd): the forward's packed words and w_scale are
bit-exact, so the backward bounds of test_gpu_train.py apply, widened by the
rstd ulp (dx and dgamma) and, for dW, by the dequantised activations
Yq = bf16(q a_scale): where the two sides' q differ, by a_scale (1 + 8u)
plus one bf16 ulp (2^-7 relative at most) of each, elsewhere by one bf16 ulp.
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
RA = 8 * U


@pytest.fixture(scope="module")
def mmf():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2406_02528_amd as m
    return m


def T_(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev())


def opt(a):
    return None if a is None else T_(a)


def chunk_len(T: int) -> int:
    return T if T <= 16 else max(16, -(-T // 128))


def sigmoid(v):
    return 1.0 / (1.0 + np.exp(-v))


def gate_bounds(z, bias, lb, flip_rows):
    """Bounds on |df|, |dc|, |dg| [M][d] from the oracle's pre-activations z
    (no bias) [M][3d]."""
    M, n3 = z.shape
    d = n3 // 3
    y = z.astype(np.float64)
    b = np.zeros(n3) if bias is None else bias.astype(np.float64)
    zz = y + b
    ref = oracle.mlgru_gates(z, bias, lb).astype(np.float64)
    low = np.zeros(d) if lb is None else lb.astype(np.float64)
    e_z = (3 * U + RA) * np.abs(y) + 2 * U * np.abs(zz)
    for s in range(3):
        seg = np.s_[s * d:(s + 1) * d]
        e_z[:, seg] += ROW_REL * np.abs(zz[:, seg]).max(axis=1, keepdims=True) * flip_rows[:, None]
    Bf = (1 - low) * e_z[:, :d] / 4 + 8 * U
    Bc = 1.1 * e_z[:, d:2 * d] + 8 * U * np.abs(ref[:, d:2 * d])
    Bg = e_z[:, 2 * d:]
    return ref, Bf, Bc, Bg


def scan_error(fcg, B, T, h0, Bf, Bc, Bg):
    """Propagated bounds on |do'_t| [B*T][d] and on |dh_T| [B][d]: the gate
    errors carried through the exact recurrence, plus the library's own
    rounding of its chunked recurrence (with magnitudes taken over the
    perturbed gates)."""
    d = fcg.shape[1] // 3
    f = fcg[:, :d].astype(np.float64).reshape(B, T, d)
    c = fcg[:, d:2 * d].astype(np.float64).reshape(B, T, d)
    g = fcg[:, 2 * d:].astype(np.float64).reshape(B, T, d)
    Bf, Bc, Bg = (a.reshape(B, T, d) for a in (Bf, Bc, Bg))
    h = np.zeros((B, d)) if h0 is None else h0.astype(np.float64)
    m = np.abs(h)
    S = np.zeros((B, d))
    D = np.zeros((B, d))
    L = chunk_len(T)
    do = np.empty((B, T, d))
    e = np.zeros((B, d))
    for t in range(T):
        ft, ct, bf, bc = f[:, t], c[:, t], Bf[:, t], Bc[:, t]
        D = ft * D + bf * (np.abs(h) + D + np.abs(ct) + bc) + (1 - ft + bf) * bc
        h = ft * h + (1 - ft) * ct
        m = np.minimum(ft + bf, 1) * m + (1 - ft + bf) * (np.abs(ct) + bc)
        S = np.minimum(ft + bf, 1) * S + m
        e = D + 2 * (L + 8) * U * S
        o = g[:, t] * sigmoid(h)
        do[:, t] = (Bg[:, t] * (sigmoid(h) + (e + U) / 4) + np.abs(g[:, t]) * (e + U) / 4 +
                    6 * U * (np.abs(o) + Bg[:, t]))
    return do.reshape(B * T, d), e


def out_proj_bounds(op_ref, dop, gamma_o, w_scale_o, t_o, b_o):
    """Bound on the output projection's error [M][N] given the oracle's o'
    and a bound dop on the library's deviation from it."""
    out = oracle.bitlinear_fwd(op_ref, gamma_o, t_o, w_scale_o)
    y = out["y"].astype(np.float64)
    o_ref = y if b_o is None else oracle.add_bias(out["y"], b_o).astype(np.float64)
    x = op_ref.astype(np.float64)
    K = x.shape[1]
    g = np.ones(K) if gamma_o is None else np.abs(gamma_o.astype(np.float64))
    xg = np.abs(x) * g
    amax = np.maximum(xg.max(axis=1, keepdims=True), 1e-30)
    # a_scale = max|o' r gamma| / 127: the maximum moves by at most the
    # largest perturbation of an element, rstd by sum |o'| dop / (sum o'^2 + K eps)
    rel_max = (dop * g).max(axis=1, keepdims=True) / amax
    rel_r = (np.abs(x) * dop).sum(axis=1, keepdims=True) / ((x * x).sum(axis=1, keepdims=True) + K * oracle.EPS)
    ra = rel_max + rel_r + RA
    # q_k = rne(127 o'_k gamma_k / max|o' gamma|) (rstd cancels): possible
    # flips where the oracle's argument lies within its movement of a midpoint
    arg = 127.0 * x * g / amax
    dist = np.abs(np.abs(arg) - np.floor(np.abs(arg)) - 0.5)
    move = 127.0 * dop * g / amax + np.abs(arg) * (ra + 4 * U)
    maybe_flip = (dist <= move).any(axis=1)
    tol = (3 * U + ra) * np.abs(y) + 2 * U * np.abs(o_ref)
    tol += ROW_REL * np.abs(y).max(axis=1, keepdims=True) * maybe_flip[:, None]
    return o_ref, tol + 1e-30, maybe_flip


MLGRU_CASES = [
    # B, T, d, bias, lb, h0, x f32
    (2, 40, 64, True, True, True, False),
    (1, 300, 32, True, False, False, False),
    (3, 1, 2048, True, True, True, False),     # decode steps: the recurrence in the output projection's prologue
    (5, 17, 48, False, True, True, True),
    (1, 1, 2048, True, True, True, False),     # the decode workload's width
]


@pytest.mark.parametrize("B,T,d,with_bias,with_lb,with_h0,f32", MLGRU_CASES)
def test_mlgru_end_to_end(mmf, B, T, d, with_bias, with_lb, with_h0, f32):
    rs = np.random.default_rng(9100 + B * 7 + T + d)
    M = B * T
    bits, xf, gamma, Wf = workloads.random_case(rs, M, d, 3 * d)
    Wo = (rs.standard_normal((d, d)) * 0.02).astype(np.float32)
    gamma_o = rs.uniform(0.5, 1.5, d).astype(np.float32)
    bias = rs.uniform(-0.5, 0.5, 3 * d).astype(np.float32) if with_bias else None
    b_o = rs.uniform(-0.5, 0.5, d).astype(np.float32) if with_bias else None
    lb = rs.uniform(0.0, 0.95, d).astype(np.float32) if with_lb else None
    h0 = (0.5 * rs.standard_normal((B, d))).astype(np.float32) if with_h0 else None
    log(f"[e2e mlgru] B={B} T={T} d={d} bias={with_bias} lb={with_lb} h0={with_h0} f32={f32}")
    # the oracle, from x alone
    tf, wsf = oracle.weight_quant(Wf)
    to, wso = oracle.weight_quant(Wo)
    ref = oracle.mlgru_fwd(xf, B, T, gamma, tf, [wsf] * 3, bias, lb, h0, gamma_o, to, wso, b_o)
    pr = oracle.mlgru_proj(xf, gamma, tf, [wsf] * 3, bias, lb)
    # the library, from x alone
    x_d = T_(xf) if f32 else to_dev_x(bits)
    Wfp, wsd = mmf.ternarize(T_(Wf))
    Wop, wsod = mmf.ternarize(T_(Wo))
    o = torch.full((M, d), float("nan"), dtype=torch.float32, device=dev())
    h_last = torch.full((B, d), float("nan"), dtype=torch.float32, device=dev())
    mmf.mmf_mlgru_fwd(x_d, B, T, T_(gamma), Wfp, torch.cat([wsd, wsd, wsd]), opt(bias), opt(lb),
                      opt(h0), h_last, T_(gamma_o), Wop, wsod, opt(b_o), o)
    q = torch.empty((M, d), dtype=torch.int8, device=dev())
    a = torch.empty((M,), dtype=torch.float32, device=dev())
    mmf.mmf_act_quant(x_d, T_(gamma), q, a)
    torch.cuda.synchronize()
    rows, _ = compare_q(q.cpu().numpy(), pr["q"])
    flip = np.zeros(M, bool)
    flip[rows] = True
    ra_in = np.abs(a.cpu().numpy().astype(np.float64) - pr["a_scale"]) / pr["a_scale"]
    assert (ra_in <= RA).all(), f"input a_scale differs by {ra_in.max():.3e} relative"
    # propagated bounds, from the oracle's values alone
    fcg_ref, Bf, Bc, Bg = gate_bounds(pr["z"], bias, lb, flip)
    assert np.array_equal(fcg_ref.astype(np.float32), ref["fcg"])
    dop, dh_last = scan_error(ref["fcg"], B, T, h0, Bf, Bc, Bg)
    o_ref, tol, maybe = out_proj_bounds(ref["o_prime"], dop, gamma_o, wso, to, b_o)
    assert np.array_equal(o_ref.astype(np.float32), ref["o"])
    got = o.cpu().numpy().astype(np.float64)
    err = np.abs(got - o_ref)
    bad = ~(err <= tol)   # NaN counts as out of bound
    assert not bad.any(), (f"o: {int(bad.sum())} out of bound (rows with a possible q flip: "
                           f"{int(maybe.sum())}), worst excess {float((err - tol).max()):.3e}")
    hg = h_last.cpu().numpy().astype(np.float64)
    err_h = np.abs(hg - ref["h_last"].astype(np.float64))
    assert not (err_h > dh_last + 1e-30).any(), f"h_last worst excess {float((err_h - dh_last).max()):.3e}"
    log(f"[e2e mlgru] rows with a possible flip in the output projection: {int(maybe.sum())}/{M}, "
        f"worst o error / bound {float((err / tol).max()):.3f}")


TRAIN_CASES = [(70, 256, 100, True), (300, 1024, 516, True), (33, 2048, 64, False)]


@pytest.mark.parametrize("M,K,N,with_gamma", TRAIN_CASES)
def test_training_step_end_to_end(mmf, M, K, N, with_gamma):
    rs = np.random.default_rng(9200 + M + K + N)
    bits, xf, gamma, W = workloads.random_case(rs, M, K, N)
    if not with_gamma:
        gamma = None
    dO_bits = workloads.f32_to_bf16_bits(rs.standard_normal((M, N)).astype(np.float32))
    dO = workloads.bf16_bits_to_f32(dO_bits)
    log(f"[e2e train] M={M} K={K} N={N} gamma={with_gamma}")
    # the oracle, from x, W and dO alone
    fw = oracle.bitlinear_train_fwd(xf, gamma, W)
    bw = oracle.bitlinear_bwd(dO, xf, gamma, fw["rstd"], fw["q"], fw["a_scale"], fw["t"], fw["w_scale"])
    # the library, from the same inputs
    x_d = to_dev_x(bits)
    g_d = None if gamma is None else T_(gamma)
    y = torch.empty((M, N), dtype=torch.float32, device=dev())
    Wp = torch.empty((K // 16, N), dtype=torch.int32, device=dev())
    ws = torch.empty((1,), dtype=torch.float32, device=dev())
    q = torch.empty((M, K), dtype=torch.int8, device=dev())
    a = torch.empty((M,), dtype=torch.float32, device=dev())
    r = torch.empty((M,), dtype=torch.float32, device=dev())
    mmf.mmf_bitlinear_train_fwd(x_d, g_d, T_(W), None, y, Wp, ws, q, a, r)
    dO_d = torch.from_numpy(dO_bits.view(np.int16)).to(dev()).view(torch.bfloat16)
    dx = torch.empty((M, K), dtype=torch.float32, device=dev())
    dW = torch.empty((N, K), dtype=torch.float32, device=dev())
    db = torch.empty((N,), dtype=torch.float32, device=dev())
    dg = torch.empty((K,), dtype=torch.float32, device=dev())
    mmf.mmf_bitlinear_bwd(dO_d, x_d, g_d, r, q, a, Wp, ws, dx, dW, db, dg if gamma is not None else None)
    torch.cuda.synchronize()
    # the forward state: words and scale bit-exact, q within the bar
    assert np.array_equal(packed_to_np(Wp), oracle.pack(fw["t"]))
    assert ws.item() == np.float32(fw["w_scale"])
    q_g = q.cpu().numpy()
    compare_q(q_g, fw["q"])
    qdiff = q_g != fw["q"]
    r_g, r_o = r.cpu().numpy().astype(np.float64), fw["rstd"].astype(np.float64)
    assert (np.abs(r_g - r_o) <= 2.0 ** -23 * r_o).all(), "rstd differs by more than 1 ulp"
    a_g = a.cpu().numpy().astype(np.float64)
    assert (np.abs(a_g - fw["a_scale"]) <= RA * fw["a_scale"]).all(), "a_scale differs"
    # bounds: the backward's own arithmetic (as test_gpu_train.py), then the
    # forward-state differences
    aO = np.abs(dO.astype(np.float64))
    x64 = xf.astype(np.float64)
    g64 = np.ones(K) if gamma is None else gamma.astype(np.float64)
    r64 = fw["rstd"].astype(np.float64)[:, None]
    w = float(fw["w_scale"])
    dY = bw["dY"]
    e1 = 2 * N * U * (aO @ np.abs(fw["t"].astype(np.float64)))
    E = w * e1 + U * np.abs(dY)
    gv = g64 * dY
    dgv = g64 * E + U * np.abs(gv)
    s = np.sum(gv * x64, axis=1, keepdims=True)
    coef = r64 ** 3 * s / K
    dcoef = r64 ** 3 / K * np.sum(dgv * np.abs(x64), axis=1, keepdims=True) + U * np.abs(coef)
    dx_ref = bw["dx"].astype(np.float64)
    rr = 2.0 ** -23  # rstd within one fp32 ulp
    tol_dx = (r64 * dgv + U * np.abs(r64 * gv) + dcoef * np.abs(x64) + U * np.abs(coef * x64) +
              U * np.abs(dx_ref) + rr * (np.abs(r64 * gv) + 3 * np.abs(coef * x64)) + 1e-30)
    yq = bw["yq"].astype(np.float64)
    a_ref = fw["a_scale"].astype(np.float64)[:, None]
    # bf16 values: one ulp is at most 2^-7 of the magnitude
    dyq = np.where(qdiff, a_ref * (1 + RA) + 2.0 ** -7 * (np.abs(yq) + a_ref), 2.0 ** -7 * np.abs(yq))
    tol_dW = 2 * M * U * (aO.T @ (np.abs(yq) + dyq)) + aO.T @ dyq + 1e-30
    tol_db = U * np.abs(aO.sum(axis=0)) + 1e-30
    for name, got, ref_v, tol in (("dx", dx, dx_ref, tol_dx), ("dW", dW, bw["dW"], tol_dW),
                                  ("db", db, bw["db"], tol_db)):
        err = np.abs(got.cpu().numpy().astype(np.float64) - ref_v.astype(np.float64))
        bad = ~(err <= tol)   # NaN counts as out of bound
        assert not bad.any(), f"{name}: {int(bad.sum())} out of bound, worst excess {float((err - tol).max()):.3e}"
    if gamma is not None:
        tol_dg = (np.sum(E * np.abs(x64) * r64, axis=0) + U * np.abs(np.sum(dY * x64 * r64, axis=0)) +
                  rr * np.sum(np.abs(dY * x64 * r64), axis=0) + 1e-30)
        err = np.abs(dg.cpu().numpy().astype(np.float64) - bw["dgamma"].astype(np.float64))
        assert (err <= tol_dg).all(), f"dgamma worst excess {float((err - tol_dg).max()):.3e}"
