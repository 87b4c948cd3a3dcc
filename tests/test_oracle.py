"""Pins for the CPU oracle: hand-worked examples, closed forms, invariants and a
second formulation of the ternary sum.  None of these re-runs the oracle's own
formula; each would fail on a dropped term, a wrong sign or index, a
transposed operand or the wrong rounding mode.  CPU only."""
import json
import math
import os

import numpy as np
import pytest

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")


@pytest.fixture(scope="module")
def golden():
    with open(GOLDEN) as f:
        return json.load(f)


# --------------------------------------------------------------------------
# hand-worked examples
# --------------------------------------------------------------------------

def test_hand_act_quant(golden):
    ex = golden["act_quant_1"]
    x = np.array([ex["x"]], np.float32)
    q, a = oracle.rmsnorm_act_quant(x, None)
    assert q[0].tolist() == ex["q"]
    _, r = oracle.rms_norm(x, None)
    assert math.isclose(float(r[0]), 1 / math.sqrt(ex["mean_square"] + 1e-6), rel_tol=1e-6)
    assert math.isclose(float(a[0]), 7 / (127 * math.sqrt(13.15625 + 1e-6)), rel_tol=1e-6)


def test_hand_act_quant_gamma(golden):
    ex = golden["act_quant_gamma"]
    x = np.array([ex["x"]], np.float32)
    g = np.array(ex["gamma"], np.float32)
    q, a = oracle.rmsnorm_act_quant(x, g)
    assert q[0].tolist() == ex["q"]
    assert math.isclose(float(a[0]), 1.6 / (127 * math.sqrt(1 + 1e-6)), rel_tol=1e-6)


def test_hand_round_half_even(golden):
    ex = golden["act_quant_ties"]
    q, a = oracle.act_quant(np.array([ex["y"]], np.float32))
    assert q[0].tolist() == ex["q"]
    assert float(a[0]) == ex["a_scale"]
    ex = golden["weight_quant_ties"]
    t, ws = oracle.weight_quant(np.array(ex["W"], np.float32))
    assert t.tolist() == ex["t"]
    assert ws == ex["w_scale"]


def test_hand_weight_quant(golden):
    ex = golden["weight_quant_1"]
    t, ws = oracle.weight_quant(np.array(ex["W"], np.float32))
    assert t.tolist() == ex["t"]
    assert math.isclose(ws, ex["w_scale"], rel_tol=1e-6)


def test_hand_accumulate(golden):
    q = np.array([golden["act_quant_1"]["q"]], np.int8)
    t = np.array(golden["weight_quant_1"]["t"], np.int8)
    acc = oracle.ternary_accumulate(q, t)
    assert acc[0].tolist() == golden["accumulate_1"]["acc"]


def test_hand_pack(golden):
    t = np.array(golden["weight_quant_1"]["t"], np.int8)
    words = oracle.pack(t)
    assert words.shape == (1, 2)
    assert [f"0x{int(w):08X}" for w in words[0]] == golden["pack_1"]["words"]
    for case in golden["pack_fixed_words"]["cases"]:
        w = oracle.pack(np.array([case["t"]], np.int8))
        assert f"0x{int(w[0, 0]):08X}" == case["word"]


# --------------------------------------------------------------------------
# weight quantisation
# --------------------------------------------------------------------------

def test_ternary_values_and_gaussian_zero_fraction():
    # For W ~ N(0, s^2), mean|W| = s sqrt(2/pi) and t = 0 iff |W| < mean/2, so
    # P(t = 0) = 2 Phi(sqrt(2/pi)/2) - 1 = erf(1 / (2 sqrt(pi))).
    w = workloads.WORKLOADS["tiny"]
    W = workloads.make_w(w)
    t, ws = oracle.weight_quant(W)
    assert set(np.unique(t).tolist()) <= {-1, 0, 1}
    p0 = math.erf(1 / (2 * math.sqrt(math.pi)))
    assert abs(p0 - 0.3101) < 1e-4
    sd = math.sqrt(p0 * (1 - p0) / t.size)
    assert abs((t == 0).mean() - p0) < 5 * sd
    # mean|N(0, 0.02^2)| = 0.02 sqrt(2/pi)
    assert abs(ws - 0.02 * math.sqrt(2 / math.pi)) < 5 * 0.02 * 0.6 / math.sqrt(t.size)
    # symmetric: +1 and -1 equally likely
    sd1 = math.sqrt(0.345 * 0.655 / t.size)
    assert abs((t == 1).mean() - (t == -1).mean()) < 7 * sd1


def test_weight_quant_power_of_two_invariance():
    rs = np.random.default_rng(1)
    W = (rs.standard_normal((33, 48)) * 0.02).astype(np.float32)
    t, ws = oracle.weight_quant(W)
    for e in (-3, 1, 4):
        t2, ws2 = oracle.weight_quant(W * np.float32(2.0 ** e))
        assert np.array_equal(t, t2)
        assert ws2 == np.float32(ws * 2.0 ** e)


def test_weight_quant_zero_tensor():
    t, ws = oracle.weight_quant(np.zeros((4, 16), np.float32))
    assert not t.any()
    assert ws == np.float32(1e-5)


def test_weight_quant_is_per_tensor():
    # scaling one row changes the codes of the other rows through the shared mean
    W = np.full((2, 16), 0.3, np.float32)
    W[0] = 1.0
    t, ws = oracle.weight_quant(W)
    assert math.isclose(ws, 0.65, rel_tol=1e-6)
    assert t[0].tolist() == [1] * 16 and t[1].tolist() == [0] * 16


# --------------------------------------------------------------------------
# packing
# --------------------------------------------------------------------------

def test_pack_roundtrip_and_invalid_code():
    rs = np.random.default_rng(2)
    t = rs.integers(-1, 2, size=(37, 64)).astype(np.int8)
    p = oracle.pack(t)
    assert p.shape == (4, 37)
    t2, bad = oracle.unpack(p, 37, 64)
    assert bad == 0 and np.array_equal(t, t2)
    p[1, 5] |= np.uint32(3 << 6)  # bits 6-7 of word j=1 hold k = 16*1 + 4*3 + 0
    t3, bad = oracle.unpack(p, 37, 64)
    assert bad == 1 and t3[5, 16 + 12] == 0


# --------------------------------------------------------------------------
# RMSNorm + activation quantisation
# --------------------------------------------------------------------------

def test_act_quant_range_and_row_max():
    rs = np.random.default_rng(3)
    x = rs.standard_normal((64, 320)).astype(np.float32)
    x[5] *= 1e-3
    x[7, 11] = 300.0
    g = rs.uniform(0.5, 1.5, 320).astype(np.float32)
    q, a = oracle.rmsnorm_act_quant(x, g)
    assert np.abs(q.astype(int)).max() <= 127
    assert (np.abs(q.astype(int)).max(axis=1) == 127).all()
    assert (q.min() >= -127)


def test_zero_row():
    x = np.zeros((2, 64), np.float32)
    x[1, 3] = 1.0
    q, a = oracle.rmsnorm_act_quant(x, None)
    assert not q[0].any()
    assert a[0] == np.float32(np.float32(1e-5) / np.float32(127.0))


@pytest.mark.parametrize("c", [3.0, -0.25, 1e-3])
def test_constant_row_closed_form(c):
    # x = c * ones, gamma = 1: mean square = c^2, so max|y| = |c| / sqrt(c^2 + eps)
    # and every q_k = 127 sign(c).  With c = 1e-3, eps = 1e-6 is as large as
    # c^2, so this also pins where eps sits and that the mean (not the sum) of
    # squares is used (K = 256).
    K = 256
    x = np.full((1, K), c, np.float32)
    q, a = oracle.rmsnorm_act_quant(x, None)
    assert (q == 127 * int(np.sign(c))).all()
    expect = abs(c) / (127 * math.sqrt(c * c + 1e-6))
    assert math.isclose(float(a[0]), expect, rel_tol=2e-6)


def test_one_hot_row():
    x = np.zeros((1, 128), np.float32)
    x[0, 17] = -4.5
    q, a = oracle.rmsnorm_act_quant(x, None)
    e = np.zeros(128, int)
    e[17] = -127
    assert np.array_equal(q[0].astype(int), e)
    # mean square = 4.5^2 / 128
    assert math.isclose(float(a[0]), 4.5 / (127 * math.sqrt(4.5 ** 2 / 128 + 1e-6)), rel_tol=2e-6)


def test_rmsnorm_scale_invariance_of_q():
    # in exact arithmetic q does not depend on r; fp32 rounding may move at
    # most a tie by one step
    rs = np.random.default_rng(4)
    x = rs.standard_normal((16, 256)).astype(np.float32)
    q1, _ = oracle.rmsnorm_act_quant(x, None)
    q2, _ = oracle.rmsnorm_act_quant(x * np.float32(3.0), None)
    d = np.abs(q1.astype(int) - q2.astype(int))
    assert d.max() <= 1 and (d > 0).mean() < 1e-2


def test_permutation_changes_q_by_at_most_one_lsb():
    rs = np.random.default_rng(5)
    x = rs.standard_normal((8, 512)).astype(np.float32)
    g = rs.uniform(0.5, 1.5, 512).astype(np.float32)
    perm = rs.permutation(512)
    q1, _ = oracle.rmsnorm_act_quant(x, g)
    q2, _ = oracle.rmsnorm_act_quant(x[:, perm], g[perm])
    d = np.abs(q1[:, perm].astype(int) - q2.astype(int))
    assert d.max() <= 1


# --------------------------------------------------------------------------
# ternary accumulation: a second formulation (integer matrix product)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("M,K,N", [(1, 16, 1), (1, 64, 17), (17, 48, 1), (5, 32, 9), (17, 64, 17)])
def test_accumulate_vs_integer_matmul(M, K, N):
    rs = np.random.default_rng(M * 1000 + K * 10 + N)
    q = rs.integers(-128, 128, size=(M, K)).astype(np.int8)
    t = rs.integers(-1, 2, size=(N, K)).astype(np.int8)
    acc = oracle.ternary_accumulate(q, t)
    ref = q.astype(np.int64) @ t.astype(np.int64).T  # multiply-add form
    assert np.array_equal(acc, ref)


def test_accumulate_special_weights():
    rs = np.random.default_rng(6)
    K = 64
    q = rs.integers(-127, 128, size=(3, K)).astype(np.int8)
    eye = np.eye(K, dtype=np.int8)
    assert np.array_equal(oracle.ternary_accumulate(q, eye), q.astype(np.int32))
    ones = np.ones((2, K), np.int8)
    s = q.astype(np.int64).sum(axis=1)
    assert np.array_equal(oracle.ternary_accumulate(q, ones), np.stack([s, s], 1))
    assert np.array_equal(oracle.ternary_accumulate(q, -ones), -np.stack([s, s], 1))
    assert not oracle.ternary_accumulate(q, np.zeros((2, K), np.int8)).any()


def test_accumulate_negation_linearity_bound():
    rs = np.random.default_rng(7)
    K = 96
    q1 = rs.integers(-60, 61, size=(4, K)).astype(np.int8)
    q2 = rs.integers(-60, 61, size=(4, K)).astype(np.int8)
    t = rs.integers(-1, 2, size=(11, K)).astype(np.int8)
    a1 = oracle.ternary_accumulate(q1, t)
    assert np.array_equal(oracle.ternary_accumulate(q1, -t), -a1)
    assert np.array_equal(oracle.ternary_accumulate((q1 + q2).astype(np.int8), t),
                          a1 + oracle.ternary_accumulate(q2, t))
    qmax = np.full((1, K), 127, np.int8)
    assert oracle.ternary_accumulate(qmax, np.ones((1, K), np.int8))[0, 0] == 127 * K


def test_accumulate_pairs_matches_full():
    rs = np.random.default_rng(8)
    q = rs.integers(-127, 128, size=(9, 80)).astype(np.int8)
    t = rs.integers(-1, 2, size=(13, 80)).astype(np.int8)
    full = oracle.ternary_accumulate(q, t)
    ms = rs.integers(0, 9, 50)
    ns = rs.integers(0, 13, 50)
    assert np.array_equal(oracle.ternary_accumulate_pairs(q, t, ms, ns), full[ms, ns])


# --------------------------------------------------------------------------
# dequantisation and the whole forward
# --------------------------------------------------------------------------

def test_fake_quant_equivalence():
    # Algorithm 1 returns fake-quantised operands round(sX)/s and round(sW)/s;
    # their fp64 product summed over k must equal the integer sum times the
    # two scales.  The fake-quant side recomputes s_a = 127/max|y| in fp64
    # from the normalised activations, so it differs from the stored fp32
    # a_scale by at most one fp32 rounding.
    rs = np.random.default_rng(9)
    x = rs.standard_normal((6, 128)).astype(np.float32)
    g = rs.uniform(0.5, 1.5, 128).astype(np.float32)
    W = (rs.standard_normal((10, 128)) * 0.02).astype(np.float32)
    t, ws = oracle.weight_quant(W)
    out = oracle.bitlinear_fwd(x, g, t, ws)
    y_norm, _ = oracle.rms_norm(x, g)
    inv_sa = np.abs(y_norm.astype(np.float64)).max(axis=1) / 127.0
    x_fq = out["q"].astype(np.float64) * inv_sa[:, None]
    w_fq = t.astype(np.float64) * ws
    o = x_fq @ w_fq.T
    rel = np.abs(out["y"] - o) / np.maximum(np.abs(o), 1e-30)
    assert rel[o != 0].max() < 3e-7
    assert (out["y"][o == 0] == 0).all()


def test_forward_negated_weights_and_zero_row():
    rs = np.random.default_rng(10)
    x = rs.standard_normal((5, 64)).astype(np.float32)
    x[2] = 0.0
    t = rs.integers(-1, 2, size=(7, 64)).astype(np.int8)
    a = oracle.bitlinear_fwd(x, None, t, 0.02)
    b = oracle.bitlinear_fwd(x, None, -t, 0.02)
    assert np.array_equal(a["y"], -b["y"])
    assert not a["y"][2].any()


def test_oracle_threads_reported():
    assert oracle.num_threads() >= 1


# --------------------------------------------------------------------------
# GLU channel-mixer gate p = SiLU(g) * u (Sec. "MatMul-free Channel Mixer")
# --------------------------------------------------------------------------

def test_glu_closed_forms():
    # sigmoid(ln 3) = 3/4 exactly, so SiLU(ln 3) = (3/4) ln 3; sigmoid(0) = 1/2.
    # A sign slip in the exponent would give ln 3 / 4 here.
    l3 = math.log(3.0)
    g = np.array([l3, -l3, 0.0, 0.0], np.float32)
    u = np.array([2.0, 2.0, 5.0, -7.0], np.float32)
    p = oracle.glu(g, u).astype(np.float64)
    g64 = float(np.float32(l3))
    assert math.isclose(p[0], 2.0 * 0.75 * g64, rel_tol=2e-7)
    assert math.isclose(p[1], 2.0 * -0.25 * g64, rel_tol=2e-7)   # SiLU(-v) = -v sigmoid(-v)
    assert p[2] == 0.0 and p[3] == 0.0


def test_glu_limits_and_odd_part():
    v = np.array([40.0, 20.0, 3.5, 1.0, 0.25], np.float32)
    one = np.ones_like(v)
    plus = oracle.glu(v, one).astype(np.float64)
    minus = oracle.glu(-v, one).astype(np.float64)
    # SiLU(v) -> v for large v, SiLU(-v) -> 0 from below
    assert plus[0] == 40.0 and abs(minus[0]) < 1e-15 and minus[0] <= 0.0
    # odd part: SiLU(v) - SiLU(-v) = v (sigmoid(v) + sigmoid(-v) = 1)
    np.testing.assert_allclose(plus - minus, v.astype(np.float64), rtol=3e-7)
    # SiLU is positive and increasing for v > 0
    assert np.all(plus > 0) and np.all(np.diff(plus[::-1]) > 0)


def test_glu_linear_in_u_and_gate_role():
    rng = np.random.default_rng(7)
    g = rng.standard_normal(64).astype(np.float32)
    u = rng.standard_normal(64).astype(np.float32)
    p = oracle.glu(g, u)
    assert np.array_equal(oracle.glu(g, 2 * u), 2 * p)          # exact: power-of-two scale
    assert np.array_equal(oracle.glu(g, -u), -p)
    assert not np.allclose(oracle.glu(u, g), p)                # the gate is the first operand
    assert np.all(oracle.glu(g, np.zeros_like(u)) == 0)


def test_glu_fwd_composition():
    # identical gate and up weights: p = SiLU(y) * y with y the BitLinear output
    rng = np.random.default_rng(3)
    x = rng.standard_normal((5, 64)).astype(np.float32)
    W = (rng.standard_normal((32, 64)) * 0.02).astype(np.float32)
    t, ws = oracle.weight_quant(W)
    out = oracle.glu_fwd(x, None, t, ws, t, ws)
    y = oracle.bitlinear_fwd(x, None, t, ws)["y"]
    assert np.array_equal(out["g"], y) and np.array_equal(out["u"], y)
    y64 = y.astype(np.float64)
    ref = y64 * y64 / (1.0 + np.exp(-y64))
    np.testing.assert_allclose(out["p"], ref, rtol=1e-6, atol=1e-30)
    # a zero activation row gives p = 0
    x[2] = 0
    assert np.all(oracle.glu_fwd(x, None, t, ws, t, ws)["p"][2] == 0)


def test_glu_interleave_blocks():
    t_g = np.arange(32 * 16, dtype=np.int32).reshape(32, 16) % 3 - 1
    t_u = (np.arange(32 * 16, dtype=np.int32).reshape(32, 16) // 7) % 3 - 1
    t = oracle.glu_interleave(t_g.astype(np.int8), t_u.astype(np.int8))
    assert t.shape == (64, 16)
    assert np.array_equal(t[0:16], t_g[0:16]) and np.array_equal(t[16:32], t_u[0:16])
    assert np.array_equal(t[32:48], t_g[16:32]) and np.array_equal(t[48:64], t_u[16:32])
    # packing the interleaved codes permutes whole columns of the separate packs
    pg, pu, pgu = oracle.pack(t_g.astype(np.int8)), oracle.pack(t_u.astype(np.int8)), oracle.pack(t)
    assert np.array_equal(pgu[:, 16:32], pu[:, 0:16]) and np.array_equal(pgu[:, 32:48], pg[:, 16:32])
    with pytest.raises(ValueError):
        oracle.glu_interleave(t_g[:24].astype(np.int8), t_u[:24].astype(np.int8))


# --------------------------------------------------------------------------
# MLGRU token mixer (Sec. "MatMul-free Language Model Architecture")
# --------------------------------------------------------------------------

def _fcg(f, c, g):
    return np.concatenate([np.asarray(f, np.float32), np.asarray(c, np.float32),
                           np.asarray(g, np.float32)], axis=-1)


def test_mlgru_gates_closed_forms():
    # sigmoid(ln 3) = 3/4 and sigmoid(0) = 1/2; with the lower bound 1/2 the
    # forget gate is 1/2 + (1/2)(3/4) = 7/8.  SiLU(ln 3) = (3/4) ln 3.
    l3 = float(np.float32(math.log(3.0)))
    z = _fcg([[l3, 0.0, -l3]], [[l3, 0.0, -l3]], [[l3, 0.0, -2.5]])
    out = oracle.mlgru_gates(z).astype(np.float64)[0]
    np.testing.assert_allclose(out[0:3], [0.75, 0.5, 0.25], rtol=2e-7)
    np.testing.assert_allclose(out[3:6], [0.75 * l3, 0.0, -0.25 * l3], rtol=2e-7)
    assert out[6:9].tolist() == [np.float32(l3), 0.0, -2.5]     # output gate: no activation
    lb = np.array([0.5, 0.5, 0.0], np.float32)
    out = oracle.mlgru_gates(z, lb=lb).astype(np.float64)[0]
    np.testing.assert_allclose(out[0:3], [0.875, 0.75, 0.25], rtol=2e-7)
    # lb = 1 pins f to 1 whatever the projection
    assert np.all(oracle.mlgru_gates(z, lb=np.ones(3, np.float32))[0, :3] == 1.0)


def test_mlgru_gates_bias_and_segments():
    rng = np.random.default_rng(11)
    d = 8
    # dyadic values: z + b is exact in fp32, so a bias equals a shifted input
    z = (rng.integers(-64, 64, (4, 3 * d)) / 16).astype(np.float32)
    b = (rng.integers(-64, 64, 3 * d) / 16).astype(np.float32)
    assert np.array_equal(oracle.mlgru_gates(z, b), oracle.mlgru_gates(z + b))
    # each segment depends on its own columns only
    base = oracle.mlgru_gates(z)
    for s in range(3):
        z2 = z.copy()
        z2[:, s * d:(s + 1) * d] += 1.0
        diff = oracle.mlgru_gates(z2) != base
        assert diff[:, s * d:(s + 1) * d].any()
        assert not np.delete(diff, np.s_[s * d:(s + 1) * d], axis=1).any()
    # sigmoid(-v) = 1 - sigmoid(v); SiLU(v) - SiLU(-v) = v
    v = np.linspace(-6, 6, d).astype(np.float32)
    zz = _fcg(v, v, v)[None]
    zn = _fcg(-v, -v, -v)[None]
    p, n = oracle.mlgru_gates(zz)[0].astype(np.float64), oracle.mlgru_gates(zn)[0].astype(np.float64)
    np.testing.assert_allclose(p[:d] + n[:d], 1.0, rtol=2e-7)
    np.testing.assert_allclose(p[d:2 * d] - n[d:2 * d], v, rtol=3e-7, atol=1e-7)
    assert np.all((p[:d] > 0) & (p[:d] < 1))


def test_mlgru_scan_constant_gates_closed_form():
    # time-invariant f and c: h_t = f^t h_0 + (1 - f^t) c (geometric series)
    T, d = 40, 5
    f = np.array([0.5, 0.9, 0.25, 0.75, 0.0], np.float32)
    c = np.array([1.0, -2.0, 3.0, 0.5, 4.0], np.float32)
    h0 = np.array([[2.0, 1.0, -1.0, 0.0, 7.0]], np.float32)
    fcg = np.tile(_fcg(f, c, np.ones(d)), (T, 1))
    o, hl = oracle.mlgru_scan(fcg, 1, T, h0)
    t = np.arange(1, T + 1)[:, None]
    f64, c64 = f.astype(np.float64), c.astype(np.float64)
    h = f64 ** t * h0.astype(np.float64) + (1 - f64 ** t) * c64
    np.testing.assert_allclose(o, 1 / (1 + np.exp(-h)), rtol=2e-7)
    np.testing.assert_allclose(hl[0], h[-1], rtol=2e-7)
    # f = 0 forgets at once (h = c), f = 1 keeps h_0 forever
    assert np.all(hl[0, 4] == 4.0)
    fcg[:, 0] = 1.0
    _, hl = oracle.mlgru_scan(fcg, 1, T, h0)
    assert hl[0, 0] == 2.0


def test_mlgru_scan_unrolled_sum():
    # second formulation: h_t = (prod_{s<=t} f_s) h_0 + sum_s (prod_{s<r<=t} f_r)(1 - f_s) c_s
    rng = np.random.default_rng(5)
    B, T, d = 2, 9, 3
    f = rng.uniform(0.05, 0.95, (B * T, d)).astype(np.float32)
    c = rng.standard_normal((B * T, d)).astype(np.float32)
    g = rng.standard_normal((B * T, d)).astype(np.float32)
    h0 = rng.standard_normal((B, d)).astype(np.float32)
    o, hl = oracle.mlgru_scan(_fcg(f, c, g), B, T, h0)
    F, C, G = (a.astype(np.float64).reshape(B, T, d) for a in (f, c, g))
    for b in range(B):
        for t in range(T):
            h = np.prod(F[b, :t + 1], axis=0) * h0[b]
            for s in range(t + 1):
                h = h + np.prod(F[b, s + 1:t + 1], axis=0) * (1 - F[b, s]) * C[b, s]
            np.testing.assert_allclose(o[b * T + t], G[b, t] / (1 + np.exp(-h)), rtol=1e-6)
        np.testing.assert_allclose(hl[b], h, rtol=1e-6)


def test_mlgru_scan_structure():
    rng = np.random.default_rng(9)
    B, T, d = 3, 12, 4
    f = rng.uniform(0.0, 1.0, (B * T, d)).astype(np.float32)
    c = rng.standard_normal((B * T, d)).astype(np.float32)
    g = rng.standard_normal((B * T, d)).astype(np.float32)
    h0 = rng.standard_normal((B, d)).astype(np.float32)
    fcg = _fcg(f, c, g)
    o, hl = oracle.mlgru_scan(fcg, B, T, h0)
    # sequences are independent: one call per sequence gives the same result
    for b in range(B):
        ob, hb = oracle.mlgru_scan(fcg[b * T:(b + 1) * T], 1, T, h0[b:b + 1])
        assert np.array_equal(ob, o[b * T:(b + 1) * T]) and np.array_equal(hb[0], hl[b])
    # no initial state is h_0 = 0; a zero candidate keeps the state at zero
    o0, _ = oracle.mlgru_scan(fcg, B, T)
    assert np.array_equal(o0, oracle.mlgru_scan(fcg, B, T, np.zeros((B, d), np.float32))[0])
    o_z, hl_z = oracle.mlgru_scan(_fcg(f, np.zeros_like(c), g), B, T)
    assert np.array_equal(o_z, g / 2) and np.all(hl_z == 0)     # sigma(0) = 1/2
    # continuing from the returned state matches one long scan (up to the fp32 state)
    t1 = 5
    oa, ha = oracle.mlgru_scan(fcg[:t1], 1, t1, h0[:1])
    ob, hb = oracle.mlgru_scan(fcg[t1:T], 1, T - t1, ha)
    np.testing.assert_allclose(np.concatenate([oa, ob]), o[:T], rtol=1e-6, atol=1e-7)
    np.testing.assert_allclose(hb[0], hl[0], rtol=1e-6, atol=1e-7)
    # linear in (h_0, c) for fixed f: the state of a sum is the sum of states
    c2 = rng.standard_normal((B * T, d)).astype(np.float32)
    h2 = rng.standard_normal((B, d)).astype(np.float32)
    big = np.full_like(g, 60.0)   # sigma(h) * 60 ~ linear readout only through h_last
    _, s1 = oracle.mlgru_scan(_fcg(f, c, big), B, T, h0)
    _, s2 = oracle.mlgru_scan(_fcg(f, c2, big), B, T, h2)
    _, s12 = oracle.mlgru_scan(_fcg(f, c + c2, big), B, T, h0 + h2)
    np.testing.assert_allclose(s12, s1.astype(np.float64) + s2, rtol=1e-5, atol=1e-6)


def test_mlgru_fwd_zero_candidate():
    # With W_c = 0 and no bias the candidate is SiLU(0) = 0, so from h_0 = 0
    # the state stays 0 and o' = g sigma(0) = g / 2.  The output projection's
    # RMSNorm removes that factor (but for eps) and absmax quantisation is
    # scale-free, so the mixer's output is BitLinear_o(g) + b_o with the same
    # q and integer sums, its scale moved only by eps.
    rng = np.random.default_rng(21)
    B, T, K = 2, 3, 32
    x = rng.standard_normal((B * T, K)).astype(np.float32)
    W = (rng.standard_normal((3 * K, K)) * 0.02).astype(np.float32)
    W[K:2 * K] = 0
    t, ws = oracle.weight_quant(W)
    Wo = (rng.standard_normal((K, K)) * 0.02).astype(np.float32)
    t_o, ws_o = oracle.weight_quant(Wo)
    b_o = (rng.integers(-8, 8, K) / 4).astype(np.float32)
    out = oracle.mlgru_fwd(x, B, T, None, t, [ws] * 3, None, None, None, None, t_o, ws_o, b_o)
    assert np.all(out["fcg"][:, K:2 * K] == 0) and np.all(out["h_last"] == 0)
    g = out["fcg"][:, 2 * K:]
    assert np.array_equal(out["o_prime"], g / 2)
    ref = oracle.bitlinear_fwd(g, None, t_o, ws_o)
    assert np.array_equal(out["q_o"], ref["q"]) and np.array_equal(out["acc_o"], ref["acc"])
    # only the RMSNorm's eps sees the factor 1/2: per row the output scale
    # is 0.5 r(g/2) / r(g) = sqrt(ms + eps) / sqrt(ms + 4 eps), ms = mean(g^2)
    ms = np.mean(g.astype(np.float64) ** 2, axis=1, keepdims=True)
    ratio = np.sqrt(ms + oracle.EPS) / np.sqrt(ms + 4 * oracle.EPS)
    assert ratio.min() < 1 - 1e-4   # the test shapes make the eps term visible
    np.testing.assert_allclose(out["o"], ref["y"].astype(np.float64) * ratio + b_o, rtol=2e-6, atol=1e-7)


def test_mlgru_proj_segment_scales():
    # segment s is scaled by w_scales[s]: doubling the candidate's scale
    # doubles exactly its pre-activations and leaves the other two alone
    rng = np.random.default_rng(23)
    K = 48
    x = rng.standard_normal((3, K)).astype(np.float32)
    t, ws = oracle.weight_quant((rng.standard_normal((3 * K, K)) * 0.02).astype(np.float32))
    p1 = oracle.mlgru_proj(x, None, t, [ws, ws, ws])
    p2 = oracle.mlgru_proj(x, None, t, [ws, 2 * ws, ws])
    assert np.array_equal(p2["z"][:, K:2 * K], 2 * p1["z"][:, K:2 * K])
    assert np.array_equal(np.delete(p2["z"], np.s_[K:2 * K], 1), np.delete(p1["z"], np.s_[K:2 * K], 1))
    assert np.array_equal(p1["acc"], oracle.ternary_accumulate(p1["q"], t))


def test_add_bias():
    y = np.array([[1.0, -2.0, 0.5]], np.float32)
    b = np.array([0.25, 2.0, -0.5], np.float32)
    assert oracle.add_bias(y, b).tolist() == [[1.25, 0.0, 0.0]]


# --------------------------------------------------------------------------
# training forward and backward (Algorithm 1, backward_pass / rms_norm_bwd;
# straight-through quantisers, Sec. "Surrogate Gradient")
# --------------------------------------------------------------------------

def _ste_case(seed, M=3, K=24, N=10, with_gamma=True):
    rs = np.random.default_rng(seed)
    x = rs.standard_normal((M, K)).astype(np.float32)
    gamma = rs.uniform(0.5, 1.5, K).astype(np.float32) if with_gamma else None
    W = (rs.standard_normal((N, K)) * 0.02).astype(np.float32)
    f = oracle.bitlinear_train_fwd(x, gamma, W)
    dO = rs.standard_normal((M, N)).astype(np.float32)
    b = oracle.bitlinear_bwd(dO, x, gamma, f["rstd"], f["q"], f["a_scale"], f["t"], f["w_scale"])
    return x, gamma, W, f, dO, b


def _surrogate(x, gamma, Wt, dO):
    """The loss the straight-through estimator differentiates: the forward with
    both quantisers replaced by the identity, sum(dO * ((x r gamma) Wt^T)),
    in fp64 with the exact rstd."""
    x = x.astype(np.float64)
    r = 1.0 / np.sqrt(np.mean(x * x, axis=1, keepdims=True) + oracle.EPS)
    y = x * r * (1.0 if gamma is None else gamma.astype(np.float64))
    return float(np.sum(dO.astype(np.float64) * (y @ Wt.T)))


@pytest.mark.parametrize("with_gamma", [True, False])
def test_bwd_dx_is_the_ste_gradient(with_gamma):
    # central differences of the surrogate loss against dx
    x, gamma, W, f, dO, b = _ste_case(31, with_gamma=with_gamma)
    Wt = f["t"].astype(np.float64) * float(f["w_scale"])
    h = 1e-4
    num = np.empty(x.shape)
    for m in range(x.shape[0]):
        for k in range(x.shape[1]):
            xp, xm = x.astype(np.float64), x.astype(np.float64)
            xp = xp.copy(); xm = xm.copy()
            xp[m, k] += h
            xm[m, k] -= h
            num[m, k] = (_surrogate(xp, gamma, Wt, dO) - _surrogate(xm, gamma, Wt, dO)) / (2 * h)
    np.testing.assert_allclose(b["dx"], num, rtol=2e-6, atol=2e-7 * np.abs(num).max())


def test_bwd_dgamma_is_the_ste_gradient():
    x, gamma, W, f, dO, b = _ste_case(32)
    Wt = f["t"].astype(np.float64) * float(f["w_scale"])
    h = 1e-4
    num = np.empty(gamma.shape)
    for k in range(gamma.size):
        gp, gm = gamma.astype(np.float64).copy(), gamma.astype(np.float64).copy()
        gp[k] += h
        gm[k] -= h
        num[k] = (_surrogate(x, gp, Wt, dO) - _surrogate(x, gm, Wt, dO)) / (2 * h)
    np.testing.assert_allclose(b["dgamma"], num, rtol=2e-6, atol=2e-7 * np.abs(num).max())


def test_bwd_dw_db_and_stored_activations():
    import torch
    x, gamma, W, f, dO, b = _ste_case(33, M=5, K=32, N=12)
    # Yq: q * a_scale in fp32, stored as bfloat16 (torch's round-to-nearest-even)
    yq = (torch.from_numpy(f["q"].astype(np.float32) * f["a_scale"][:, None])
          .to(torch.bfloat16).to(torch.float32).numpy())
    assert np.array_equal(b["yq"], yq)
    # the loss is linear in the forward's weights Wt: its gradient is dO^T Yq
    np.testing.assert_allclose(b["dW"], dO.astype(np.float64).T @ yq.astype(np.float64), rtol=1e-6, atol=1e-7)
    np.testing.assert_allclose(b["db"], dO.astype(np.float64).sum(axis=0), rtol=1e-6, atol=1e-7)


def test_bwd_invariant_pins_eps():
    # sum_k x_k dx_k = eps r^3 s exactly (s = sum_k gamma_k dY_k x_k): the
    # normalisation's gradient is orthogonal to x up to the eps term
    x, gamma, W, f, dO, b = _ste_case(34, M=4, K=48, N=8)
    r = f["rstd"].astype(np.float64)
    s = np.sum(gamma.astype(np.float64) * b["dY"] * x, axis=1)
    lhs = np.sum(x.astype(np.float64) * b["dx"], axis=1)
    scale = np.abs(r * s) * 1e-6 + 1e-12
    assert np.all(np.abs(lhs - oracle.EPS * r ** 3 * s) <= scale)
    # zero output gradient: zero everywhere
    z = oracle.bitlinear_bwd(np.zeros_like(dO), x, gamma, f["rstd"], f["q"], f["a_scale"], f["t"], f["w_scale"])
    assert not z["dx"].any() and not z["dW"].any() and not z["db"].any() and not z["dgamma"].any()


def test_train_fwd_rstd_and_bias():
    rs = np.random.default_rng(35)
    x = rs.standard_normal((4, 64)).astype(np.float32)
    W = (rs.standard_normal((16, 64)) * 0.02).astype(np.float32)
    b = (rs.integers(-8, 8, 16) / 8).astype(np.float32)
    f = oracle.bitlinear_train_fwd(x, None, W, b)
    r = 1.0 / np.sqrt(np.mean(x.astype(np.float64) ** 2, axis=1) + 1e-6)
    np.testing.assert_allclose(f["rstd"], r, rtol=1e-7)
    f0 = oracle.bitlinear_train_fwd(x, None, W)
    np.testing.assert_allclose(f["y"], f0["y"].astype(np.float64) + b, rtol=1e-7, atol=1e-7)


def test_bwd_bf16_storage_rounds_ties_to_even():
    # q * a_scale = +-(1 + 2^-8) lies halfway between the bf16 values 1
    # (mantissa even) and 1 + 2^-7 (odd): ties to even give 1
    a = np.array([1 + 2.0 ** -8, 1 + 2.0 ** -7 + 2.0 ** -8], np.float32)
    q = np.array([[1, -1], [1, -1]], np.int8)
    K, N = 2, 1
    b = oracle.bitlinear_bwd(np.zeros((2, N), np.float32), np.ones((2, K), np.float32), None,
                             np.ones(2, np.float32), q, a, np.zeros((N, K), np.int8), 1.0)
    assert b["yq"][0].tolist() == [1.0, -1.0]
    # 1 + 3 * 2^-8 = 1 + 1.5 * 2^-7: between mantissas 1 (odd) and 2 (even)
    assert b["yq"][1].tolist() == [1.015625, -1.015625]
