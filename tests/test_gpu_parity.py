"""GPU parity: the HIP path through the C ABI against the CPU oracle on the
same seeded inputs.  Integer results are compared bit for bit; fp32 results
with the tolerances in tests/_parity.py."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from _parity import (Case, compare_q, compare_y, dev, log, np_to_packed, packed_to_np,
                     to_dev_x)

pytestmark = pytest.mark.gpu

PATHS = ("gemv", "gemm")


@pytest.fixture(scope="module")
def mmf():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2406_02528_amd as m
    return m


def set_path(mmf, name):
    return mmf.mmf_set_path({"auto": 0, "gemv": 1, "gemm": 2}[name])


def run_forward(mmf, case, Wp, ws, path):
    prev = set_path(mmf, path)
    try:
        y = torch.full((case.M, case.N), float("nan"), dtype=torch.float32, device=dev())
        mmf.mmf_bitlinear_fwd(case.x_d, case.g_d, Wp, ws, y)
        torch.cuda.synchronize()
    finally:
        mmf.mmf_set_path(prev)
    return y


def run_i32(mmf, q_d, Wp, M, N, path):
    prev = set_path(mmf, path)
    try:
        acc = torch.full((M, N), -(2 ** 31), dtype=torch.int32, device=dev())
        mmf.mmf_ternary_gemm_i32(q_d, Wp, acc)
        torch.cuda.synchronize()
    finally:
        mmf.mmf_set_path(prev)
    return acc


def gpu_weights(mmf, case):
    Wp, ws = mmf.ternarize(case.W_d)
    torch.cuda.synchronize()
    return Wp, ws


def check_weights(case, Wp, ws):
    words = packed_to_np(Wp)
    assert words.shape == case.words_ref.shape
    assert np.array_equal(words, case.words_ref), \
        f"{int((words != case.words_ref).sum())} packed words differ"
    assert float(ws.item()) == case.ws_ref, (float(ws.item()), case.ws_ref)


def gpu_act(mmf, case):
    q = torch.empty((case.M, case.K), dtype=torch.int8, device=dev())
    a = torch.empty((case.M,), dtype=torch.float32, device=dev())
    rs = torch.empty((case.M,), dtype=torch.int32, device=dev())
    mmf.mmf_act_quant(case.x_d, case.g_d, q, a, rs)
    torch.cuda.synchronize()
    return q, a, rs


def check_act(case, q, a, rs):
    qn = q.cpu().numpy()
    flip_rows, frac = compare_q(qn, case.q_ref)
    an = a.cpu().numpy()
    same = np.ones(case.M, bool)
    same[flip_rows] = False
    rel = np.abs(an[same].astype(np.float64) - case.a_ref[same]) / case.a_ref[same]
    assert rel.max(initial=0) <= 1e-6
    assert np.array_equal(rs.cpu().numpy(), qn.astype(np.int64).sum(axis=1))
    return qn, flip_rows, frac


# ---------------------------------------------------------------------------
# full-size comparisons on the small workloads
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("wl", ["tiny", "decode_m1", "decode_m8"])
def test_workload_full(mmf, wl):
    w = workloads.WORKLOADS[wl]
    log(f"[{wl}] M={w.M} K={w.K} N={w.N}: inputs + oracle")
    case = Case.from_workload(w)
    case.oracle_weights()
    case.oracle_act()
    acc_ref = oracle.ternary_accumulate(case.q_ref, case.t)
    y_ref = oracle.dequant(acc_ref, case.a_ref, case.ws_ref)
    case.upload()
    log(f"[{wl}] ternarize")
    Wp, ws = gpu_weights(mmf, case)
    check_weights(case, Wp, ws)
    log(f"[{wl}] act_quant")
    q, a, rs = gpu_act(mmf, case)
    qn, flip_rows, _ = check_act(case, q, a, rs)
    flip_mask = np.zeros(case.M, bool)
    flip_mask[flip_rows] = True
    q_ref_d = torch.from_numpy(case.q_ref).to(dev())
    for path in PATHS:
        log(f"[{wl}] i32 contraction, {path}")
        acc = run_i32(mmf, q_ref_d, Wp, case.M, case.N, path).cpu().numpy()
        assert np.array_equal(acc, acc_ref), f"{path}: {int((acc != acc_ref).sum())} sums differ"
        log(f"[{wl}] forward, {path}")
        y = run_forward(mmf, case, Wp, ws, path).cpu().numpy()
        compare_y(y, y_ref, acc_ref, flip_mask)


# ---------------------------------------------------------------------------
# full-size prefill workloads: full packed words and q, sampled outputs
# ---------------------------------------------------------------------------

def sample_pairs(rs, M, N, P=4096):
    ms = rs.integers(0, M, P)
    ns = rs.integers(0, N, P)
    corners_m = np.array([0, 0, M - 1, M - 1])
    corners_n = np.array([0, N - 1, 0, N - 1])
    return np.concatenate([ms, corners_m]), np.concatenate([ns, corners_n])


@pytest.mark.parametrize("wl", ["glu_up", "glu_down", "large", "large_dec"])
def test_workload_sampled(mmf, wl):
    w = workloads.WORKLOADS[wl]
    log(f"[{wl}] M={w.M} K={w.K} N={w.N}: inputs + oracle")
    case = Case.from_workload(w)
    case.oracle_weights()
    case.oracle_act()
    case.upload()
    log(f"[{wl}] ternarize")
    Wp, ws = gpu_weights(mmf, case)
    check_weights(case, Wp, ws)
    del case.W_d
    log(f"[{wl}] act_quant")
    q, a, rs_ = gpu_act(mmf, case)
    qn, flip_rows, frac = check_act(case, q, a, rs_)
    log(f"[{wl}] q flips: {frac:.2e}")
    rs = np.random.default_rng(w.index)
    ms, ns = sample_pairs(rs, case.M, case.N)
    acc_ref = oracle.ternary_accumulate_pairs(case.q_ref, case.t, ms, ns)
    y_ref = (acc_ref.astype(np.float64) * case.a_ref[ms].astype(np.float64) *
             np.float64(case.ws_ref)).astype(np.float32)
    ms_d = torch.from_numpy(ms).to(dev())
    ns_d = torch.from_numpy(ns).to(dev())
    log(f"[{wl}] i32 contraction (auto path)")
    q_ref_d = torch.from_numpy(case.q_ref).to(dev())
    acc = run_i32(mmf, q_ref_d, Wp, case.M, case.N, "auto")
    got = acc[ms_d, ns_d].cpu().numpy()
    del acc
    assert np.array_equal(got, acc_ref), f"{int((got != acc_ref).sum())} sampled sums differ"
    log(f"[{wl}] forward (auto path)")
    y = run_forward(mmf, case, Wp, ws, "auto")
    assert not torch.isnan(y).any().item(), "forward left outputs unwritten"
    got_y = y[ms_d, ns_d].cpu().numpy()
    flip_mask = np.isin(ms, flip_rows)
    compare_y(got_y[:, None], y_ref[:, None], acc_ref[:, None], flip_mask)
    # whole rows 0 and M-1 against the oracle
    for m in (0, case.M - 1):
        full_ref = oracle.ternary_accumulate(case.q_ref[m:m + 1], case.t)
        yr = oracle.dequant(full_ref, case.a_ref[m:m + 1], case.ws_ref)
        compare_y(y[m:m + 1].cpu().numpy(), yr, full_ref, np.array([m in flip_rows]))


# ---------------------------------------------------------------------------
# small random shapes through both kernels (ragged tiles, K tails, N tails)
# ---------------------------------------------------------------------------

SWEEP_M = [1, 2, 3, 5, 8, 9, 15, 16, 17, 33, 257]
SWEEP_K = [16, 48, 64, 256, 2064]
SWEEP_N = [1, 16, 64, 257, 1024]


def check_shape(mmf, rs, M, K, N, paths, tag="sweep"):
    """One random case: weights and act-quant against the oracle, then the
    exact int32 sums and the forward through each of `paths`."""
    bits, xf, g, W = workloads.random_case(rs, M, K, N)
    case = Case(bits, xf, g, W, f"M{M}K{K}N{N}")
    case.oracle_weights()
    case.oracle_act()
    acc_ref = oracle.ternary_accumulate(case.q_ref, case.t)
    y_ref = oracle.dequant(acc_ref, case.a_ref, case.ws_ref)
    case.upload()
    log(f"[{tag}] M={M} K={K} N={N}")
    Wp, ws = gpu_weights(mmf, case)
    check_weights(case, Wp, ws)
    q, a, r = gpu_act(mmf, case)
    qn, flip_rows, _ = check_act(case, q, a, r)
    flip = np.zeros(M, bool)
    flip[flip_rows] = True
    q_ref_d = torch.from_numpy(case.q_ref).to(dev())
    for path in paths:
        acc = run_i32(mmf, q_ref_d, Wp, M, N, path).cpu().numpy()
        assert np.array_equal(acc, acc_ref), (path, M, K, N)
        y = run_forward(mmf, case, Wp, ws, path).cpu().numpy()
        assert not np.isnan(y).any(), ("forward left outputs unwritten", path, M, K, N)
        compare_y(y, y_ref, acc_ref, flip)


@pytest.mark.parametrize("M", SWEEP_M)
def test_random_shapes(mmf, M):
    rs = np.random.default_rng(1000 + M)
    for K in SWEEP_K:
        for N in SWEEP_N:
            check_shape(mmf, rs, M, K, N, PATHS)


# The MFMA kernel's tile shape follows the problem (on 256 compute units):
# 64 x 256 tiles for a short M or a narrow N, 64 x 512 in between, 128 x 512
# once the wide tiles fill the CUs, run as two 128 x 256 workgroups per CU at
# K <= 4096 beyond one round of wide tiles (the full-size workloads above
# take both forms).  Ragged in every dimension (a partial last stage of K,
# partial row and column tiles).  The automatic path sends 33-64 tokens to
# the MFMA kernel at K <= 2048 and to decode launches of 16 tokens beyond.
@pytest.mark.parametrize("M,K,N", [(300, 1040, 2000),    # 64 x 256: 40 tiles
                                   (1000, 336, 6000),    # 64 x 512: 192 tiles
                                   (1100, 528, 8000),    # 128 x 512: 144 tiles, one round
                                   (3000, 400, 8200),    # 128 x 256 pairs: 816 tiles
                                   (40, 2048, 1000),     # auto: MFMA kernel (64 x 256)
                                   (57, 2064, 1000)])    # auto: four decode launches
def test_gemm_tile_shapes(mmf, M, K, N):
    check_shape(mmf, np.random.default_rng(1100 + M + K), M, K, N, PATHS + ("auto",), tag="tiles")


# ---------------------------------------------------------------------------
# degenerate inputs and buffer discipline
# ---------------------------------------------------------------------------

def test_degenerate_rows_and_weights(mmf):
    M, K, N = 12, 256, 96
    rs = np.random.default_rng(7)
    x = rs.standard_normal((M, K)).astype(np.float32)
    x[1] = 0.0                      # zero row -> q = 0, y = 0
    x[2] = 0.75                     # constant row -> q = 127
    x[3] = 0.0
    x[3, 5] = -3.0                  # one-hot row
    x[4] *= 1e-30                   # tiny row: eps dominates, the 1e-5 absmax floor applies
    W = (rs.standard_normal((N, K)) * 0.02).astype(np.float32)
    W[7] = 0.0                      # a zero output column
    case = Case(x, x, None, W, "degenerate")
    case.oracle_weights()
    case.oracle_act()
    case.upload()
    log("[degenerate] f32 rows")
    Wp, ws = gpu_weights(mmf, case)
    check_weights(case, Wp, ws)
    q, a, r = gpu_act(mmf, case)
    qn, _, _ = check_act(case, q, a, r)
    assert not qn[1].any() and (qn[2] == 127).all()
    acc_ref = oracle.ternary_accumulate(case.q_ref, case.t)
    y_ref = oracle.dequant(acc_ref, case.a_ref, case.ws_ref)
    for path in PATHS:
        y = run_forward(mmf, case, Wp, ws, path).cpu().numpy()
        compare_y(y, y_ref, acc_ref)
        assert not y[1].any() and not y[:, 7].any()


def test_all_zero_weights(mmf):
    W = torch.zeros((64, 128), dtype=torch.float32, device=dev())
    log("[zero weights]")
    Wp, ws = mmf.ternarize(W)
    torch.cuda.synchronize()
    assert float(ws.item()) == np.float32(1e-5)
    assert (packed_to_np(Wp) == 0x55555555).all()


def test_empty_shapes_leave_outputs_untouched(mmf):
    log("[empty shapes]")
    x = torch.zeros((0, 64), dtype=torch.bfloat16, device=dev())
    Wp = torch.zeros((4, 32), dtype=torch.int32, device=dev())
    ws = torch.ones(1, device=dev())
    y = torch.zeros((0, 32), device=dev())
    mmf.mmf_bitlinear_fwd(x, None, Wp, ws, y)
    x2 = torch.zeros((3, 64), dtype=torch.bfloat16, device=dev())
    y2 = torch.zeros((3, 0), device=dev())
    mmf.mmf_bitlinear_fwd(x2, None, torch.zeros((4, 0), dtype=torch.int32, device=dev()), ws, y2)
    torch.cuda.synchronize()


def test_guard_bands_and_determinism(mmf):
    """Outputs written into the middle of larger buffers leave the guard bands
    untouched, and two runs give identical bits."""
    M, K, N = 37, 272, 300
    rs = np.random.default_rng(11)
    bits, xf, g, W = workloads.random_case(rs, M, K, N)
    case = Case(bits, xf, g, W, "guard")
    case.upload()
    Wp, ws = gpu_weights(mmf, case)
    G = 1024
    for path in PATHS:
        log(f"[guard] {path}")
        prev = set_path(mmf, path)
        try:
            outs = []
            for _ in range(2):
                buf = torch.full((G + M * N + G,), 12345.0, device=dev())
                y = buf[G:G + M * N].view(M, N)
                mmf.mmf_bitlinear_fwd(case.x_d, case.g_d, Wp, ws, y)
                torch.cuda.synchronize()
                assert (buf[:G] == 12345.0).all() and (buf[G + M * N:] == 12345.0).all()
                outs.append(y.clone())
            assert torch.equal(outs[0], outs[1])
        finally:
            mmf.mmf_set_path(prev)
    # act_quant guard bands
    qbuf = torch.full((G + M * K + G,), 77, dtype=torch.int8, device=dev())
    q = qbuf[G:G + M * K].view(M, K)
    a = torch.empty(M, device=dev())
    mmf.mmf_act_quant(case.x_d, case.g_d, q, a)
    torch.cuda.synchronize()
    assert (qbuf[:G] == 77).all() and (qbuf[G + M * K:] == 77).all()


def test_workspace_variant_matches(mmf):
    w = workloads.WORKLOADS["decode_m8"]
    case = Case.from_workload(w)
    case.upload()
    Wp, ws = gpu_weights(mmf, case)
    log("[workspace variant]")
    y1 = torch.empty((case.M, case.N), device=dev())
    mmf.mmf_bitlinear_fwd(case.x_d, case.g_d, Wp, ws, y1)
    nbytes = mmf.mmf_bitlinear_workspace_bytes(case.M, case.K)
    wsb = torch.empty(nbytes, dtype=torch.uint8, device=dev())
    y2 = torch.empty_like(y1)
    mmf.mmf_bitlinear_fwd_ws(case.x_d, case.g_d, Wp, ws, y2, wsb)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)


def test_dequant_entry_matches_forward(mmf):
    w = workloads.WORKLOADS["tiny"]
    case = Case.from_workload(w)
    case.upload()
    Wp, ws = gpu_weights(mmf, case)
    log("[gemm_dequant entry]")
    q, a, r = gpu_act(mmf, case)
    for path in PATHS:
        prev = set_path(mmf, path)
        try:
            y1 = torch.empty((case.M, case.N), device=dev())
            mmf.mmf_ternary_gemm_dequant(q, a, r, Wp, ws, y1)
            y2 = torch.empty_like(y1)
            mmf.mmf_bitlinear_fwd(case.x_d, case.g_d, Wp, ws, y2)
            torch.cuda.synchronize()
            assert torch.equal(y1, y2)
        finally:
            mmf.mmf_set_path(prev)


@pytest.mark.parametrize("M,K,N", [(8, 8192, 300), (3, 24576, 70), (1, 32768, 129)])
def test_decode_fallback_shapes(mmf, M, K, N):
    """Decode shapes whose quantised rows do not fit the fused kernel's LDS
    take the two-launch path (act-quant kernel + global-q contraction)."""
    rs = np.random.default_rng(M * 7 + K)
    bits, xf, g, W = workloads.random_case(rs, M, K, N)
    case = Case(bits, xf, g, W, f"fallback M{M}K{K}N{N}")
    case.oracle_weights()
    case.oracle_act()
    acc_ref = oracle.ternary_accumulate(case.q_ref, case.t)
    y_ref = oracle.dequant(acc_ref, case.a_ref, case.ws_ref)
    case.upload()
    log(f"[fallback] M={M} K={K} N={N}")
    Wp, ws = gpu_weights(mmf, case)
    check_weights(case, Wp, ws)
    q, a, r = gpu_act(mmf, case)
    qn, flip_rows, _ = check_act(case, q, a, r)
    flip = np.zeros(M, bool)
    flip[flip_rows] = True
    acc = run_i32(mmf, torch.from_numpy(case.q_ref).to(dev()), Wp, M, N, "auto").cpu().numpy()
    assert np.array_equal(acc, acc_ref)
    y = run_forward(mmf, case, Wp, ws, "auto").cpu().numpy()
    compare_y(y, y_ref, acc_ref, flip)


@pytest.mark.parametrize("M,K,N,f32", [(1, 4096, 324, False), (2, 4112, 1000, False), (1, 8192, 96, True),
                                       (2, 5120, 15360, False), (1, 4608, 4, True)])
def test_decode_large_blocks(mmf, M, K, N, f32):
    """Decode shapes with many word rows per workgroup (eight weight loads in
    flight per lane, or more in groups of eight): ragged column tails
    (N % 64 != 0), K/16 not a multiple of 4 (the last step's missing word
    rows read as zero), bf16 and fp32 activations, and through the affine
    epilogue (a bias)."""
    rs = np.random.default_rng(M * 13 + K + N)
    bits, xf, g, W = workloads.random_case(rs, M, K, N)
    x_form = xf if f32 else bits
    case = Case(x_form, xf, g, W, f"lds M{M}K{K}N{N}")
    case.oracle_weights()
    case.oracle_act()
    acc_ref = oracle.ternary_accumulate(case.q_ref, case.t)
    y_ref = oracle.dequant(acc_ref, case.a_ref, case.ws_ref)
    case.upload()
    log(f"[decode large blocks] M={M} K={K} N={N} f32={f32}")
    Wp, ws = gpu_weights(mmf, case)
    check_weights(case, Wp, ws)
    q, a, r = gpu_act(mmf, case)
    qn, flip_rows, _ = check_act(case, q, a, r)
    flip = np.zeros(M, bool)
    flip[flip_rows] = True
    y = run_forward(mmf, case, Wp, ws, "auto").cpu().numpy()
    compare_y(y, y_ref, acc_ref, flip)
    # the same shape under the affine epilogue: y + b must equal the plain
    # forward plus b, rounded once more
    b = rs.uniform(-0.5, 0.5, N).astype(np.float32)
    yb = torch.empty((M, N), dtype=torch.float32, device=dev())
    mmf.mmf_bitlinear_fwd_bias(case.x_d, case.g_d, Wp, ws, torch.from_numpy(b).to(dev()), yb)
    yp = run_forward(mmf, case, Wp, ws, "auto")
    torch.cuda.synchronize()
    expect = (yp.cpu().numpy().astype(np.float32) + b).astype(np.float32)
    assert np.array_equal(yb.cpu().numpy(), expect)


@pytest.mark.parametrize("M,K,N,f32", [(4, 1040, 9000, False), (3, 2048, 8194, False), (3, 8192, 2000, False),
                                       (5, 1024, 1000, True), (8, 4096, 640, False), (2, 2064, 6146, True)])
def test_decode_matrix_core_layouts(mmf, M, K, N, f32):
    """Two to eight tokens are contracted on the matrix cores inside the fused
    decode kernel.  Column blocks of 16 per workgroup: four with 16-byte
    weight loads (N = 9000), two (N = 6146), two because N % 4 != 0 although
    the grid then exceeds one round of CUs (N = 8194), one (the rest).  K/16
    not a multiple of 4 (the last k64 step masks its missing word rows, and
    waves past K/16 hold no step), more k64 steps per wave than are in flight
    at once (K = 8192), the largest bf16 row set (8 x 4096), fp32
    activations; the integer hook from pre-quantised q (padded LDS rows when
    K % 1024 == 0, unpadded otherwise) and the affine epilogue (N % 4 == 0)."""
    rs = np.random.default_rng(M * 31 + K + N)
    bits, xf, g, W = workloads.random_case(rs, M, K, N)
    x_form = xf if f32 else bits
    case = Case(x_form, xf, g, W, f"mfma M{M}K{K}N{N}")
    case.oracle_weights()
    case.oracle_act()
    acc_ref = oracle.ternary_accumulate(case.q_ref, case.t)
    y_ref = oracle.dequant(acc_ref, case.a_ref, case.ws_ref)
    case.upload()
    log(f"[decode mfma] M={M} K={K} N={N} f32={f32}")
    Wp, ws = gpu_weights(mmf, case)
    check_weights(case, Wp, ws)
    q, a, r = gpu_act(mmf, case)
    qn, flip_rows, _ = check_act(case, q, a, r)
    flip = np.zeros(M, bool)
    flip[flip_rows] = True
    acc = run_i32(mmf, torch.from_numpy(case.q_ref).to(dev()), Wp, M, N, "auto").cpu().numpy()
    assert np.array_equal(acc, acc_ref)
    y = run_forward(mmf, case, Wp, ws, "auto").cpu().numpy()
    compare_y(y, y_ref, acc_ref, flip)
    if N % 4 == 0:  # the entry point with a bias takes N % 4 == 0 only
        b = rs.uniform(-0.5, 0.5, N).astype(np.float32)
        yb = torch.empty((M, N), dtype=torch.float32, device=dev())
        mmf.mmf_bitlinear_fwd_bias(case.x_d, case.g_d, Wp, ws, torch.from_numpy(b).to(dev()), yb)
        torch.cuda.synchronize()
        expect = (y.astype(np.float32) + b).astype(np.float32)
        assert np.array_equal(yb.cpu().numpy(), expect)


@pytest.mark.parametrize("M,K,N,f32", [(9, 2048, 6144, False), (15, 2064, 1000, False), (16, 2048, 6144, False),
                                       (16, 1024, 520, True), (12, 4096, 640, False), (16, 7680, 192, False),
                                       (33, 2048, 2048, False), (40, 1040, 96, True)])
def test_decode_up_to_16_tokens_per_launch(mmf, M, K, N, f32):
    """Nine to sixteen tokens run as one launch of the decode kernel (all 16
    rows of the matrix-core operand carry tokens; rows past M read as zero):
    9, 15 and 16 tokens fused from x; 12 x 4096 and 16 x 7680, whose rows
    need more registers than the fused kernel holds, from act-quant's q
    copied into LDS (16 x 7680 is the largest q region); 33 and 40 tokens as
    launches of 16, 16 and the rest on the forced decode path (the automatic
    path sends more than 32 tokens at K <= 2048 to the MFMA kernel)."""
    rs = np.random.default_rng(M * 17 + K + N)
    bits, xf, g, W = workloads.random_case(rs, M, K, N)
    x_form = xf if f32 else bits
    case = Case(x_form, xf, g, W, f"dec16 M{M}K{K}N{N}")
    case.oracle_weights()
    case.oracle_act()
    acc_ref = oracle.ternary_accumulate(case.q_ref, case.t)
    y_ref = oracle.dequant(acc_ref, case.a_ref, case.ws_ref)
    case.upload()
    log(f"[decode 16] M={M} K={K} N={N} f32={f32}")
    Wp, ws = gpu_weights(mmf, case)
    check_weights(case, Wp, ws)
    q, a, r = gpu_act(mmf, case)
    qn, flip_rows, _ = check_act(case, q, a, r)
    flip = np.zeros(M, bool)
    flip[flip_rows] = True
    for path in ("auto", "gemv"):
        acc = run_i32(mmf, torch.from_numpy(case.q_ref).to(dev()), Wp, M, N, path).cpu().numpy()
        assert np.array_equal(acc, acc_ref), path
        y = run_forward(mmf, case, Wp, ws, path).cpu().numpy()
        compare_y(y, y_ref, acc_ref, flip)
