"""GPU parity of the training forward and the backward of the BitLinear
(Algorithm 1, forward_pass with the latent weights quantised per call;
backward_pass and rms_norm_bwd in the RMSNorm reading, straight-through
quantisers per Sec. "Surrogate Gradient") through the C ABI, against the CPU
oracle on the same seeded inputs.

Bars, with u = 2^-24:
  * training forward: packed words and w_scale bit-exact, rstd within 1 ulp
    (fp64 sums of squares in different orders); q within the
    activation-quantisation bar; y as the inference forward (with a bias:
    (3u + r_a)|y| + 2u|y + b|, r_a the measured relative a_scale difference);
  * backward, on the GPU forward's own q, a_scale and rstd (the forward is
    checked above): the two products are bf16 GEMMs whose products of bf16
    values are exact in fp32, so any order of fp32 accumulation keeps
    |error| <= (n - 1) u sum|terms|; the test allows 2 n u sum|terms| (n the
    contraction length) for dW and for dY before the weight scale, then
    propagates: dY = fp32(w dYs) adds u|dY|, g = gamma dY adds u|g|,
    s = sum g x (fp64) inherits sum |dg||x|, coef = r^3 s / K adds u|coef|,
    and dx = r g - coef x adds u on each of its three roundings;
    db (fp64 sums of bf16 values, rounded once) within u|db|; dgamma
    (fp64 sums of fp32(w dYs) x r) within sum |dY error| |x| r + u|dgamma|.
  * integer-valued output gradients make dY exact (sums of small integers in
    fp32): that case is held to the rounding terms alone.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from _parity import compare_q, compare_y, dev, log, packed_to_np, to_dev_x

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


@pytest.fixture(scope="module")
def mmf():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2406_02528_amd as m
    return m


def T_(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev())


def bf16_tensor(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev()).view(torch.bfloat16)


def train_fwd_gpu(mmf, x_d, g_d, W, bias):
    M, K = x_d.shape
    N = W.shape[0]
    y = torch.full((M, N), float("nan"), dtype=torch.float32, device=dev())
    Wp = torch.empty((K // 16, N), dtype=torch.int32, device=dev())
    ws = torch.empty((1,), dtype=torch.float32, device=dev())
    q = torch.empty((M, K), dtype=torch.int8, device=dev())
    a = torch.empty((M,), dtype=torch.float32, device=dev())
    r = torch.empty((M,), dtype=torch.float32, device=dev())
    mmf.mmf_bitlinear_train_fwd(x_d, g_d, T_(W), None if bias is None else T_(bias), y, Wp, ws, q, a, r)
    torch.cuda.synchronize()
    return {"y": y, "Wp": Wp, "ws": ws, "q": q, "a": a, "r": r}


@pytest.mark.parametrize("M,K,N,with_bias", [(1, 16, 4, False), (5, 64, 36, True), (70, 256, 100, False),
                                             (300, 1024, 516, True)])
def test_train_fwd(mmf, M, K, N, with_bias):
    rs = np.random.default_rng(8000 + M + N)
    bits, xf, gamma, W = workloads.random_case(rs, M, K, N)
    bias = rs.uniform(-0.5, 0.5, N).astype(np.float32) if with_bias else None
    log(f"[train fwd] M={M} K={K} N={N} bias={with_bias}")
    g = train_fwd_gpu(mmf, to_dev_x(bits), T_(gamma), W, bias)
    ref = oracle.bitlinear_train_fwd(xf, gamma, W, bias)
    assert np.array_equal(packed_to_np(g["Wp"]), oracle.pack(ref["t"]))
    assert g["ws"].item() == np.float32(ref["w_scale"])
    # rstd: both sides round 1/sqrt(mean + eps) from an fp64 sum of squares
    # taken in different orders: within one fp32 ulp
    r_g, r_o = g["r"].cpu().numpy().astype(np.float64), ref["rstd"].astype(np.float64)
    assert (np.abs(r_g - r_o) <= 2.0 ** -23 * r_o).all(), "rstd differs by more than 1 ulp"
    flip_rows, _ = compare_q(g["q"].cpu().numpy(), ref["q"])
    mask = np.zeros(M, bool)
    mask[flip_rows] = True
    y = g["y"].cpu().numpy()
    if bias is None:
        compare_y(y, ref["y"], ref["acc"], mask)
    else:
        y0 = oracle.bitlinear_fwd(xf, gamma, ref["t"], ref["w_scale"])["y"].astype(np.float64)
        a_ref = ref["a_scale"].astype(np.float64)
        ra = np.abs(g["a"].cpu().numpy() - a_ref) / a_ref
        out = ref["y"].astype(np.float64)
        tol = (3 * U + ra[:, None]) * np.abs(y0) + 2 * U * np.abs(out) + 1e-30
        tol += 1e-3 * np.abs(y0).max(axis=1, keepdims=True) * mask[:, None]
        assert (np.abs(y - out) <= tol).all()


def bwd_bounds(dO, x, gamma, r, t, ws, yq, dY, exact_dy: bool):
    """Per-element bounds (dx, dW, db, dgamma) for the library's arithmetic,
    from the oracle's fp64 dY and the inputs."""
    M, N = dO.shape
    K = x.shape[1]
    aO = np.abs(dO.astype(np.float64))
    x64 = x.astype(np.float64)
    g = np.ones(K) if gamma is None else gamma.astype(np.float64)
    r64 = r.astype(np.float64)[:, None]
    w = float(ws)
    e1 = 0.0 if exact_dy else 2 * N * U * (aO @ np.abs(t.astype(np.float64)))   # dYs before w
    E = w * e1 + U * np.abs(dY)                                                  # dy = fp32(w dYs)
    gv = g * dY
    dg = g * E + U * np.abs(gv)
    s = np.sum(gv * x64, axis=1, keepdims=True)
    coef = r64 ** 3 * s / K
    dcoef = r64 ** 3 / K * np.sum(dg * np.abs(x64), axis=1, keepdims=True) + U * np.abs(coef)
    dx_ref = r64 * gv - coef * x64
    tol_dx = r64 * dg + U * np.abs(r64 * gv) + dcoef * np.abs(x64) + U * np.abs(coef * x64) + U * np.abs(dx_ref)
    tol_dW = 2 * M * U * (aO.T @ np.abs(yq.astype(np.float64)))
    tol_db = U * np.abs(aO.sum(axis=0)) + 1e-30
    tol_dg = np.sum(E * np.abs(x64) * r64, axis=0) + U * np.abs(np.sum(dY * x64 * r64, axis=0))
    return tol_dx + 1e-30, tol_dW + 1e-30, tol_db, tol_dg + 1e-30


def check(name, got, ref, tol):
    err = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    bad = ~(err <= tol)   # NaN counts as out of bound
    if bad.any():
        i = np.unravel_index(np.argmax(err - tol), err.shape)
        raise AssertionError(f"{name}: {int(bad.sum())} out of bound; worst at {i}: got {got[i]!r} "
                             f"ref {ref[i]!r} tol {tol[i]:.3e}")


def run_bwd(mmf, M, K, N, f32_x, with_gamma, int_grad=False, seed=0, dgamma=True, db=True):
    rs = np.random.default_rng(seed)
    bits, xf, gamma, W = workloads.random_case(rs, M, K, N)
    if not with_gamma:
        gamma = None
    x_host = xf if f32_x else bits
    x_d = to_dev_x(x_host)
    g_d = None if gamma is None else T_(gamma)
    fw = train_fwd_gpu(mmf, x_d, g_d, W, None)
    t, ws = oracle.weight_quant(W)
    assert np.array_equal(packed_to_np(fw["Wp"]), oracle.pack(t))
    if int_grad:
        dO_f = rs.integers(-8, 9, (M, N)).astype(np.float32)
    else:
        dO_f = rs.standard_normal((M, N)).astype(np.float32)
    dO_bits = workloads.f32_to_bf16_bits(dO_f)
    dO_f = workloads.bf16_bits_to_f32(dO_bits)
    dx = torch.full((M, K), float("nan"), dtype=torch.float32, device=dev())
    dW = torch.full((N, K), float("nan"), dtype=torch.float32, device=dev())
    dbt = torch.full((N,), float("nan"), dtype=torch.float32, device=dev()) if db else None
    dgt = torch.full((K,), float("nan"), dtype=torch.float32, device=dev()) if dgamma else None
    mmf.mmf_bitlinear_bwd(bf16_tensor(dO_bits), x_d, g_d, fw["r"], fw["q"], fw["a"], fw["Wp"], fw["ws"],
                          dx, dW, dbt, dgt)
    torch.cuda.synchronize()
    q, a, r = fw["q"].cpu().numpy(), fw["a"].cpu().numpy(), fw["r"].cpu().numpy()
    ref = oracle.bitlinear_bwd(dO_f, xf, gamma, r, q, a, t, ws)
    tdx, tdW, tdb, tdg = bwd_bounds(dO_f, xf, gamma, r, t, ws, ref["yq"], ref["dY"], int_grad)
    check("dx", dx.cpu().numpy(), ref["dx"], tdx)
    check("dW", dW.cpu().numpy(), ref["dW"], tdW)
    if db:
        check("db", dbt.cpu().numpy(), ref["db"], tdb)
    if dgamma:
        check("dgamma", dgt.cpu().numpy(), ref["dgamma"], tdg)
    return dx, dW, dbt, dgt


@pytest.mark.parametrize("M,K,N", [(1, 16, 1), (5, 64, 36), (70, 256, 100), (300, 1024, 513),
                                   (33, 2048, 40), (17, 4096, 24),   # rows held in registers / re-read
                                   (4096, 256, 128)])                # dW split over tokens
@pytest.mark.parametrize("f32_x,with_gamma", [(False, True), (True, False)])
def test_bwd_random(mmf, M, K, N, f32_x, with_gamma):
    log(f"[bwd] M={M} K={K} N={N} f32_x={f32_x} gamma={with_gamma}")
    run_bwd(mmf, M, K, N, f32_x, with_gamma, seed=9000 + M + K + N + 7 * f32_x)


def test_bwd_integer_gradients_exact_products(mmf):
    log("[bwd] integer-valued dO")
    run_bwd(mmf, 129, 512, 200, False, True, int_grad=True, seed=9100)


def test_bwd_optional_outputs_and_workspace(mmf):
    # leaving db and dgamma out changes nothing else; caller workspace gives the same bits
    dx1, dW1, _, _ = run_bwd(mmf, 33, 128, 48, False, True, seed=9200)
    dx2, dW2, _, _ = run_bwd(mmf, 33, 128, 48, False, True, seed=9200, db=False, dgamma=False)
    assert torch.equal(dx1, dx2) and torch.equal(dW1, dW2)


@pytest.mark.parametrize("M,K,N", [(1000, 2288, 3998),    # 144 dW tiles: all of them spread over 256 units
                                   (1000, 3840, 5120)])   # 300 tiles: 256 whole, 44 spread over 88 units
def test_bwd_dw_tail_pieces(mmf, M, K, N):
    """dW with more output tiles than half the compute units (256 on MI355X):
    whole tiles take the full rounds of workgroups and the stages of the
    remaining tiles are spread evenly over one more round, in pieces that a
    unit may take from two tiles and that a second kernel adds.  dW is checked
    against the oracle on every output row of the first and the last (ragged)
    256-row tile and on one row of every other, so each tile is covered;
    dx on sampled token rows; db on the sampled columns."""
    log(f"[bwd tail] M={M} K={K} N={N}")
    rs = np.random.default_rng(9300 + N)
    bits, xf, gamma, W = workloads.random_case(rs, M, K, N)
    x_d, g_d = to_dev_x(bits), T_(gamma)
    fw = train_fwd_gpu(mmf, x_d, g_d, W, None)
    t, ws = oracle.weight_quant(W)
    assert np.array_equal(packed_to_np(fw["Wp"]), oracle.pack(t))
    dO_bits = workloads.f32_to_bf16_bits(rs.standard_normal((M, N)).astype(np.float32))
    dO_f = workloads.bf16_bits_to_f32(dO_bits)
    dx = torch.full((M, K), float("nan"), dtype=torch.float32, device=dev())
    dW = torch.full((N, K), float("nan"), dtype=torch.float32, device=dev())
    db = torch.full((N,), float("nan"), dtype=torch.float32, device=dev())
    mmf.mmf_bitlinear_bwd(bf16_tensor(dO_bits), x_d, g_d, fw["r"], fw["q"], fw["a"], fw["Wp"], fw["ws"],
                          dx, dW, db, None)
    torch.cuda.synchronize()
    q, a, r = fw["q"].cpu().numpy(), fw["a"].cpu().numpy(), fw["r"].cpu().numpy()
    rows = np.unique(np.concatenate([rs.integers(0, M, 40), [0, M - 1]]))
    ref = oracle.bitlinear_bwd(dO_f[rows], xf[rows], gamma, r[rows], q[rows], a[rows], t, ws)
    tdx, _, _, _ = bwd_bounds(dO_f[rows], xf[rows], gamma, r[rows], t, ws, ref["yq"], ref["dY"], False)
    check("dx (sampled rows)", dx.cpu().numpy()[rows], ref["dx"], tdx)
    last = (N - 1) // 256 * 256
    one_per_tile = [rs.integers(n0, min(n0 + 256, N)) for n0 in range(256, last, 256)]
    cols = np.unique(np.concatenate([np.arange(0, 256), one_per_tile, np.arange(last, N)]))
    ref = oracle.bitlinear_bwd(dO_f[:, cols], xf, gamma, r, q, a, t[cols], ws)
    _, tdW, tdb, _ = bwd_bounds(dO_f[:, cols], xf, gamma, r, t[cols], ws, ref["yq"], ref["dY"], False)
    check("dW (output rows)", dW.cpu().numpy()[cols], ref["dW"], tdW)
    check("db (sampled)", db.cpu().numpy()[cols], ref["db"], tdb)


@pytest.mark.parametrize("name", ["train_d1024", "train_glu_up"])
def test_train_workload_full_size_sampled(mmf, name):
    """The paper's training-efficiency setting (input size and sequence length
    1024; 16 sequences, M = 16384, K = N = 1024; its dW has 16 output tiles, so
    every tile's token range is split) and the 1.3B model's GLU up-projection
    over 8192 tokens (352 dW tiles: 256 whole, the stages of the other 96
    spread evenly over 256 more units and their pieces added by a second
    kernel): training
    forward and backward at full size; dx rows and dW rows sampled from two
    oracle calls (rows of tokens, then columns of outputs), db sampled."""
    w = workloads.TRAIN_WORKLOADS[name]
    inp = workloads.make_train(w)
    log(f"[{name}] M={w.M} K={w.K} N={w.N}")
    x_d, g_d = to_dev_x(inp["x_bits"]), T_(inp["gamma"])
    fw = train_fwd_gpu(mmf, x_d, g_d, inp["W"], None)
    t, ws = oracle.weight_quant(inp["W"])
    assert np.array_equal(packed_to_np(fw["Wp"]), oracle.pack(t))
    dO_f = workloads.bf16_bits_to_f32(inp["dO_bits"])
    dx = torch.empty((w.M, w.K), dtype=torch.float32, device=dev())
    dW = torch.empty((w.N, w.K), dtype=torch.float32, device=dev())
    db = torch.empty((w.N,), dtype=torch.float32, device=dev())
    mmf.mmf_bitlinear_bwd(bf16_tensor(inp["dO_bits"]), x_d, g_d, fw["r"], fw["q"], fw["a"], fw["Wp"],
                          fw["ws"], dx, dW, db, None)
    torch.cuda.synchronize()
    q, a, r = fw["q"].cpu().numpy(), fw["a"].cpu().numpy(), fw["r"].cpu().numpy()
    xf = inp["x_f32"]
    rs = np.random.default_rng(10)
    rows = np.unique(np.concatenate([rs.integers(0, w.M, 60), [0, w.M - 1]]))
    ref = oracle.bitlinear_bwd(dO_f[rows], xf[rows], inp["gamma"], r[rows], q[rows], a[rows], t, ws)
    tdx, _, _, _ = bwd_bounds(dO_f[rows], xf[rows], inp["gamma"], r[rows], t, ws, ref["yq"], ref["dY"], False)
    check("dx (sampled rows)", dx.cpu().numpy()[rows], ref["dx"], tdx)
    cols = np.unique(np.concatenate([rs.integers(0, w.N, 30), [0, w.N - 1]]))
    ref = oracle.bitlinear_bwd(dO_f[:, cols], xf, inp["gamma"], r, q, a, t[cols], ws)
    _, tdW, tdb, _ = bwd_bounds(dO_f[:, cols], xf, inp["gamma"], r, t[cols], ws, ref["yq"], ref["dY"], False)
    check("dW (sampled output rows)", dW.cpu().numpy()[cols], ref["dW"], tdW)
    check("db (sampled)", db.cpu().numpy()[cols], ref["db"], tdb)
