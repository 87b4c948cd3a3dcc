"""GPU parity of the fused GLU up-projection and gate (Sec. "MatMul-free
Channel Mixer": g = x (*) W_g, u = x (*) W_u, p = SiLU(g) * u) through the C
ABI, against the CPU oracle on the same seeded inputs.

Bar:
  * interleaved packed words: bit-exact against the oracle's own packing of
    its interleaved codes;
  * p: the library's g and u are the BitLinear outputs (within 2 fp32 ulps of
    the oracle's, which rounds an fp64 product once), and SiLU(g) * u
    magnifies a relative error of g by at most 1 + |g| sigmoid(-g) <= 1 + |g|;
    for |g| < 32 that keeps p within ~1e-5 relative.  The test asks for
    |dp| <= 1e-3 |p_ref| per element on rows whose int8 activations match
    exactly, plus an absolute 1e-6 max|p_ref| (over the row) for the SiLU tail
    at large negative g where p underflows towards 0; p == 0 exactly where the
    gate or the up sum is 0; rows with an activation LSB flip use
    max|dp| <= 1e-3 max|p_ref| over the row.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from _parity import Case, compare_q, dev, log, packed_to_np

pytestmark = pytest.mark.gpu

P_REL = 1e-3
P_TAIL_ABS = 1e-6


@pytest.fixture(scope="module")
def mmf():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2406_02528_amd as m
    return m


def compare_p(p_gpu, p_ref, acc_g, acc_u, flip_rows_mask):
    p_gpu = p_gpu.astype(np.float64)
    p_ref = p_ref.astype(np.float64)
    err = np.abs(p_gpu - p_ref)
    rowmax = np.abs(p_ref).max(axis=1, keepdims=True)
    ok = ~flip_rows_mask
    zero = (acc_g == 0) | (acc_u == 0)
    assert (p_gpu[ok][zero[ok]] == 0).all(), "nonzero p where a ternary sum is 0"
    bound = P_REL * np.abs(p_ref) + P_TAIL_ABS * rowmax
    bad = ~(err <= bound) & ok[:, None]   # NaN counts as out of bound
    assert not bad.any(), f"{int(bad.sum())} p values out of bound, worst {float((err - bound).max()):.3e}"
    for m in np.nonzero(flip_rows_mask)[0]:
        assert err[m].max(initial=0.0) <= P_REL * rowmax[m, 0] + 1e-30
    nz = (p_ref != 0) & ok[:, None]
    return float((err[nz] / np.abs(p_ref[nz])).max(initial=0.0))


def gpu_pack(mmf, W_g, W_u, joint: bool):
    """Ternarise gate and up (jointly: one scale over [W_g; W_u]; else each its
    own) and interleave.  Returns (Wgu, w_scales tensor, t_g, t_u, ws_g, ws_u)."""
    L, K = W_g.shape
    if joint:
        W = np.concatenate([W_g, W_u], axis=0)
        t, ws = oracle.weight_quant(W)
        t_g, t_u, ws_g, ws_u = t[:L], t[L:], ws, ws
        Wp, wsd = mmf.ternarize(torch.from_numpy(W).to(dev()))
        Wg_p = Wp[:, :L].contiguous()
        Wu_p = Wp[:, L:].contiguous()
        w_scales = torch.cat([wsd, wsd])
    else:
        t_g, ws_g = oracle.weight_quant(W_g)
        t_u, ws_u = oracle.weight_quant(W_u)
        Wg_p, wsg = mmf.ternarize(torch.from_numpy(W_g).to(dev()))
        Wu_p, wsu = mmf.ternarize(torch.from_numpy(W_u).to(dev()))
        w_scales = torch.cat([wsg, wsu])
    Wgu = mmf.glu_pack(Wg_p, Wu_p)
    torch.cuda.synchronize()
    words_ref = oracle.pack(oracle.glu_interleave(t_g, t_u))
    assert np.array_equal(packed_to_np(Wgu), words_ref), "interleaved packed words differ"
    assert w_scales.cpu().numpy().tolist() == [np.float32(ws_g), np.float32(ws_u)]
    return Wgu, w_scales, t_g, t_u, ws_g, ws_u


def test_glu_paired_tiles_ragged(mmf):
    """A shape whose GLU contraction runs as two 128 x 256 workgroups per CU
    (408 wide tiles, more than one round, at K <= 4096), ragged in every
    dimension: 3000 = 23 * 128 + 56 tokens, 2 L = 8224 = 32 * 256 + 32
    interleaved columns, K = 400 = 3 * 128 + 16 (a whole ring period, then a
    partial stage with the offsets set afresh)."""
    M, K, L = 3000, 400, 4112
    rs = np.random.default_rng(2400)
    bits, xf, g, W = workloads.random_case(rs, M, K, 2 * L)
    log(f"[glu paired tiles] M={M} K={K} L={L}")
    Wgu, w_scales, t_g, t_u, ws_g, ws_u = gpu_pack(mmf, W[:L], W[L:], False)
    ref = oracle.glu_fwd(xf, g, t_g, ws_g, t_u, ws_u)
    case = Case(bits, xf, g, W, "")
    case.upload()
    q = torch.empty((M, K), dtype=torch.int8, device=dev())
    a = torch.empty((M,), dtype=torch.float32, device=dev())
    mmf.mmf_act_quant(case.x_d, case.g_d, q, a)
    p = torch.full((M, L), float("nan"), dtype=torch.float32, device=dev())
    mmf.mmf_glu_fwd(case.x_d, case.g_d, Wgu, w_scales, p)
    torch.cuda.synchronize()
    flip_rows, _ = compare_q(q.cpu().numpy(), ref["q"])
    flip = np.zeros(M, bool)
    flip[flip_rows] = True
    compare_p(p.cpu().numpy(), ref["p"], ref["acc_g"], ref["acc_u"], flip)


@pytest.mark.parametrize("M", [1, 8, 17, 300])
def test_glu_random_shapes(mmf, M):
    rs = np.random.default_rng(2000 + M)
    for K in (16, 64, 2064):
        for L in (16, 48, 160):
            joint = bool((K + L) % 2)
            bits, xf, g, W = workloads.random_case(rs, M, K, 2 * L)
            log(f"[glu] M={M} K={K} L={L} joint={joint}")
            Wgu, w_scales, t_g, t_u, ws_g, ws_u = gpu_pack(mmf, W[:L], W[L:], joint)
            ref = oracle.glu_fwd(xf, g, t_g, ws_g, t_u, ws_u)
            case = Case(bits, xf, g, W, "")
            case.upload()
            q = torch.empty((M, K), dtype=torch.int8, device=dev())
            a = torch.empty((M,), dtype=torch.float32, device=dev())
            mmf.mmf_act_quant(case.x_d, case.g_d, q, a)
            p = torch.full((M, L), float("nan"), dtype=torch.float32, device=dev())
            mmf.mmf_glu_fwd(case.x_d, case.g_d, Wgu, w_scales, p)
            torch.cuda.synchronize()
            flip_rows, _ = compare_q(q.cpu().numpy(), ref["q"])
            flip = np.zeros(M, bool)
            flip[flip_rows] = True
            compare_p(p.cpu().numpy(), ref["p"], ref["acc_g"], ref["acc_u"], flip)


def test_glu_workspace_variant_matches(mmf):
    rs = np.random.default_rng(77)
    M, K, L = 33, 256, 64
    bits, xf, g, W = workloads.random_case(rs, M, K, 2 * L)
    Wgu, w_scales, *_ = gpu_pack(mmf, W[:L], W[L:], True)
    case = Case(bits, xf, g, W, "")
    case.upload()
    p1 = mmf.glu(case.x_d, case.g_d, Wgu, w_scales)
    ws = torch.empty(mmf.mmf_bitlinear_workspace_bytes(M, K), dtype=torch.uint8, device=dev())
    p2 = torch.empty_like(p1)
    mmf.mmf_glu_fwd_ws(case.x_d, case.g_d, Wgu, w_scales, p2, ws)
    # the contraction stage alone, from the quantised activations
    q = torch.empty((M, K), dtype=torch.int8, device=dev())
    a = torch.empty((M,), dtype=torch.float32, device=dev())
    r = torch.empty((M,), dtype=torch.int32, device=dev())
    mmf.mmf_act_quant(case.x_d, case.g_d, q, a, r)
    p3 = torch.empty_like(p1)
    mmf.mmf_ternary_gemm_glu(q, a, r, Wgu, w_scales, p3)
    torch.cuda.synchronize()
    assert torch.equal(p1, p2) and torch.equal(p1, p3)


def test_glu_up_full_size_sampled(mmf):
    """The GLU up-projection shape (M=8192, K=2048, L=5632, bf16 x with 1%
    outlier channels), gate|up ternarised jointly as the concatenated
    projection: full packed words and q, sampled p, whole first/last rows."""
    w = workloads.WORKLOADS["glu_up"]
    L = w.N // 2
    log(f"[glu_up] M={w.M} K={w.K} L={L}: inputs + oracle")
    case = Case.from_workload(w)
    case.oracle_act()
    Wgu, w_scales, t_g, t_u, ws_g, ws_u = gpu_pack(mmf, case.W[:L], case.W[L:], True)
    case.upload()
    del case.W_d
    q = torch.empty((case.M, case.K), dtype=torch.int8, device=dev())
    a = torch.empty((case.M,), dtype=torch.float32, device=dev())
    mmf.mmf_act_quant(case.x_d, case.g_d, q, a)
    log("[glu_up] forward")
    p = torch.full((case.M, L), float("nan"), dtype=torch.float32, device=dev())
    mmf.mmf_glu_fwd(case.x_d, case.g_d, Wgu, w_scales, p)
    torch.cuda.synchronize()
    assert not torch.isnan(p).any().item(), "outputs left unwritten"
    flip_rows, frac = compare_q(q.cpu().numpy(), case.q_ref)
    log(f"[glu_up] q flips: {frac:.2e}")
    rs = np.random.default_rng(5)
    ms = np.concatenate([rs.integers(0, case.M, 4096), [0, 0, case.M - 1, case.M - 1]])
    cs = np.concatenate([rs.integers(0, L, 4096), [0, L - 1, 0, L - 1]])
    acc_g = oracle.ternary_accumulate_pairs(case.q_ref, t_g, ms, cs)
    acc_u = oracle.ternary_accumulate_pairs(case.q_ref, t_u, ms, cs)
    g_ref = oracle.dequant(acc_g[:, None], case.a_ref[ms], ws_g)
    u_ref = oracle.dequant(acc_u[:, None], case.a_ref[ms], ws_u)
    p_ref = oracle.glu(g_ref, u_ref)
    got = p[torch.from_numpy(ms).to(dev()), torch.from_numpy(cs).to(dev())].cpu().numpy()[:, None]
    flip = np.isin(ms, flip_rows)
    # sampled pairs are independent one-element rows: the tail term uses |p_ref| itself
    compare_p(got, p_ref, acc_g[:, None], acc_u[:, None], flip)
    for m in (0, case.M - 1):
        ref = oracle.glu_fwd(case.x_f32[m:m + 1], case.gamma, t_g, ws_g, t_u, ws_u)
        compare_p(p[m:m + 1].cpu().numpy(), ref["p"], ref["acc_g"], ref["acc_u"],
                  np.array([m in flip_rows]))


@pytest.mark.parametrize("M,K,L,f32", [(1, 2064, 48, False), (1, 4096, 160, False), (3, 1024, 1024, False),
                                       (8, 2048, 4160, False), (17, 256, 16, True), (40, 512, 5632, False),
                                       (2, 4096, 1040, True)])
def test_glu_decode_epilogue(mmf, M, K, L, f32):
    """Few tokens take the fused decode kernel with the GLU epilogue (launches
    of at most 8 tokens): one token on the vector ALU with 32- or 64-column
    workgroups (and the LDS-staged weights at K = 4096), two to eight on the
    matrix cores with two or four 16-column blocks per workgroup, several
    slices, bf16 and fp32 x.  p against the oracle, and bit for bit against
    the MFMA kernel's GLU epilogue."""
    rs = np.random.default_rng(3000 + M + K + L)
    bits, xf, g, W = workloads.random_case(rs, M, K, 2 * L)
    x_form = xf if f32 else bits
    Wgu, w_scales, t_g, t_u, ws_g, ws_u = gpu_pack(mmf, W[:L], W[L:], bool((K + L) % 2))
    ref = oracle.glu_fwd(xf, g, t_g, ws_g, t_u, ws_u)
    case = Case(x_form, xf, g, W, "")
    case.upload()
    log(f"[glu decode] M={M} K={K} L={L} f32={f32}")
    outs = []
    for path in (mmf.MMF_PATH_GEMV, mmf.MMF_PATH_GEMM):
        prev = mmf.mmf_set_path(path)
        try:
            p = torch.full((M, L), float("nan"), dtype=torch.float32, device=dev())
            mmf.mmf_glu_fwd(case.x_d, case.g_d, Wgu, w_scales, p)  # bf16 or fp32 x by dtype
            torch.cuda.synchronize()
        finally:
            mmf.mmf_set_path(prev)
        outs.append(p.cpu().numpy())
    q = torch.empty((M, K), dtype=torch.int8, device=dev())
    a = torch.empty((M,), dtype=torch.float32, device=dev())
    mmf.mmf_act_quant(case.x_d, case.g_d, q, a)
    torch.cuda.synchronize()
    flip_rows, _ = compare_q(q.cpu().numpy(), ref["q"])
    flip = np.zeros(M, bool)
    flip[flip_rows] = True
    compare_p(outs[0], ref["p"], ref["acc_g"], ref["acc_u"], flip)
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
