"""C-ABI checks that need no GPU: the library loads, exports every function
that include/mmf.h declares, and its host-side argument checks reject bad
calls before anything is enqueued (no pointer is dereferenced on these paths,
so stand-in addresses are used)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mmf.h")


@pytest.fixture(scope="module")
def mmf():
    import paper_2406_02528_amd as m
    return m


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mmf_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("mmf_ternarize_weights", "mmf_act_quant", "mmf_bitlinear_fwd",
                     "mmf_ternary_gemm_i32"):
        assert required in names


def test_library_exports_every_declared_symbol(mmf):
    lib = ctypes.CDLL(mmf.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings_and_sizes(mmf):
    assert mmf.mmf_version() >= 1
    assert mmf.mmf_status_string(0) == "MMF_OK"
    for s in range(1, 8):
        assert mmf.mmf_status_string(s).startswith("MMF_ERR")
    assert "DTYPE" in mmf.mmf_status_string(4) and "HIP" in mmf.mmf_status_string(5)
    assert "WORKSPACE" in mmf.mmf_status_string(6)
    assert "unknown" in mmf.mmf_status_string(99)
    assert mmf.mmf_packed_weight_bytes(6144, 2048) == 6144 * 2048 // 4
    assert mmf.mmf_packed_weight_bytes(3, 48) == 3 * 3 * 4
    assert mmf.mmf_packed_weight_bytes(3, 40) == 0   # K % 16 != 0
    assert mmf.mmf_packed_weight_bytes(3, 0) == 0
    ws = mmf.mmf_bitlinear_workspace_bytes(8192, 2048)
    assert ws >= 8192 * 2048 + 8 * 8192 and ws % 256 == 0
    assert mmf.mmf_bitlinear_workspace_bytes(1, 17) == 0


def test_set_path(mmf):
    prev = mmf.mmf_set_path(mmf.MMF_PATH_GEMV)
    assert mmf.mmf_set_path(mmf.MMF_PATH_GEMM) == mmf.MMF_PATH_GEMV
    assert mmf.mmf_set_path(prev) == mmf.MMF_PATH_GEMM
    with pytest.raises(ValueError):
        mmf.mmf_set_path(7)


A = 0x10000      # 16-byte aligned stand-in device addresses, never dereferenced
B = 0x20000
C = 0x30000
D = 0x40000
E = 0x50000
BAD = 0x10004    # 4-byte aligned only
S = None         # null stream


def _c(mmf):
    return mmf._lib


@pytest.mark.parametrize("K", [0, -16, 8, 24, 2 ** 20 + 16])
def test_bad_k_is_rejected(mmf, K):
    lib = _c(mmf)
    assert lib.mmf_bitlinear_fwd(A, B, C, D, E, 4, K, 4, S) == 2
    assert lib.mmf_act_quant(A, B, C, D, 4, K, S) == 2
    assert lib.mmf_act_quant_ex(A, 0, B, C, D, E, 4, K, S) == 2
    assert lib.mmf_ternarize_weights(A, 4, K, B, C, S) == 2
    assert lib.mmf_ternary_gemm_i32(A, B, C, 4, K, 4, S) == 2
    assert lib.mmf_ternary_gemm_dequant(A, B, C, D, E, A, 4, K, 4, S) == 2


def test_bad_m_n_are_rejected(mmf):
    lib = _c(mmf)
    assert lib.mmf_bitlinear_fwd(A, B, C, D, E, -1, 16, 4, S) == 2
    assert lib.mmf_bitlinear_fwd(A, B, C, D, E, 4, 16, 2 ** 31, S) == 2
    assert lib.mmf_ternarize_weights(A, -5, 16, B, C, S) == 2


def test_null_pointers(mmf):
    lib = _c(mmf)
    assert lib.mmf_bitlinear_fwd(None, B, C, D, E, 4, 16, 4, S) == 1
    assert lib.mmf_bitlinear_fwd(A, B, None, D, E, 4, 16, 4, S) == 1
    assert lib.mmf_bitlinear_fwd(A, B, C, None, E, 4, 16, 4, S) == 1
    assert lib.mmf_bitlinear_fwd(A, B, C, D, None, 4, 16, 4, S) == 1
    assert lib.mmf_act_quant(A, None, None, D, 4, 16, S) == 1
    assert lib.mmf_act_quant(A, None, C, None, 4, 16, S) == 1
    assert lib.mmf_act_quant_f32(None, None, C, D, 4, 16, S) == 1
    assert lib.mmf_ternarize_weights(None, 4, 16, B, C, S) == 1
    assert lib.mmf_ternarize_weights(A, 4, 16, B, None, S) == 1
    assert lib.mmf_ternary_gemm_i32(A, None, C, 4, 16, 4, S) == 1
    assert lib.mmf_ternary_gemm_dequant(A, B, None, D, E, A, 4, 16, 4, S) == 1
    assert lib.mmf_bitlinear_fwd_ws(A, 0, B, C, D, E, 4, 16, 4, None, 1 << 20, S) == 1


def test_misaligned_pointers(mmf):
    lib = _c(mmf)
    assert lib.mmf_bitlinear_fwd(BAD, B, C, D, E, 4, 16, 4, S) == 3
    assert lib.mmf_bitlinear_fwd(A, BAD, C, D, E, 4, 16, 4, S) == 3
    assert lib.mmf_bitlinear_fwd(A, B, BAD, D, E, 4, 16, 4, S) == 3
    assert lib.mmf_bitlinear_fwd(A, B, C, D, BAD, 4, 16, 4, S) == 3
    assert lib.mmf_act_quant(A, B, BAD, D, 4, 16, S) == 3
    assert lib.mmf_act_quant_ex(A, 0, B, C, D, BAD, 4, 16, S) == 3
    assert lib.mmf_ternarize_weights(BAD, 4, 16, B, C, S) == 3
    assert lib.mmf_ternary_gemm_i32(A, B, BAD, 4, 16, 4, S) == 3


def test_workspace_checks(mmf):
    lib = _c(mmf)
    need = mmf.mmf_bitlinear_workspace_bytes(4, 16)
    assert lib.mmf_bitlinear_fwd_ws(A, 0, B, C, D, E, 4, 16, 4, 0x100000, need - 1, S) == 6
    assert lib.mmf_bitlinear_fwd_ws(A, 0, B, C, D, E, 4, 16, 4, 0x100010, need, S) == 6
    assert lib.mmf_bitlinear_fwd_ws(A, 2, B, C, D, E, 4, 16, 4, 0x100000, need, S) == 4


def test_empty_shapes_are_noops(mmf):
    # M == 0 or N == 0 returns OK without touching (or even checking) buffers
    lib = _c(mmf)
    assert lib.mmf_bitlinear_fwd(None, None, None, None, None, 0, 16, 4, S) == 0
    assert lib.mmf_bitlinear_fwd(None, None, None, None, None, 4, 16, 0, S) == 0
    assert lib.mmf_act_quant(None, None, None, None, 0, 16, S) == 0
    assert lib.mmf_ternarize_weights(None, 0, 16, None, None, S) == 0
    assert lib.mmf_ternary_gemm_i32(None, None, None, 0, 16, 5, S) == 0


def test_python_binding_rejects_cpu_tensors(mmf):
    import torch
    x = torch.zeros(2, 16, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        mmf.mmf_act_quant(x, None, torch.zeros(2, 16, dtype=torch.int8), torch.zeros(2))
    with pytest.raises(TypeError):
        mmf.mmf_act_quant(torch.zeros(2, 16, dtype=torch.float16), None,
                          torch.zeros(2, 16, dtype=torch.int8), torch.zeros(2))


def test_glu_argument_checks(mmf):
    lib = _c(mmf)
    # L must be a multiple of 16; K as for the forward
    assert lib.mmf_glu_fwd(A, B, C, D, E, 4, 16, 24, S) == 2
    assert lib.mmf_glu_fwd(A, B, C, D, E, 4, 24, 32, S) == 2
    assert lib.mmf_glu_fwd(A, B, C, D, E, 4, 16, -16, S) == 2
    assert lib.mmf_glu_pack(A, B, 24, 16, C, S) == 2
    assert lib.mmf_glu_pack(A, B, 32, 40, C, S) == 2
    # NULL and misaligned pointers
    assert lib.mmf_glu_fwd(None, B, C, D, E, 4, 16, 32, S) == 1
    assert lib.mmf_glu_fwd(A, B, C, None, E, 4, 16, 32, S) == 1
    assert lib.mmf_glu_fwd(A, B, C, D, None, 4, 16, 32, S) == 1
    assert lib.mmf_glu_fwd(A, B, BAD, D, E, 4, 16, 32, S) == 3
    assert lib.mmf_glu_fwd_f32(A, B, C, D, BAD, 4, 16, 32, S) == 3
    assert lib.mmf_glu_pack(A, None, 32, 16, C, S) == 1
    assert lib.mmf_glu_pack(A, B, 32, 16, BAD, S) == 3
    # workspace variant
    need = mmf.mmf_bitlinear_workspace_bytes(4, 16)
    assert lib.mmf_glu_fwd_ws(A, 0, B, C, D, E, 4, 16, 32, 0x100000, need - 1, S) == 6
    assert lib.mmf_glu_fwd_ws(A, 0, B, C, D, E, 4, 16, 32, None, need, S) == 1
    assert lib.mmf_glu_fwd_ws(A, 3, B, C, D, E, 4, 16, 32, 0x100000, need, S) == 4
    # empty shapes are no-ops
    assert lib.mmf_glu_fwd(None, None, None, None, None, 0, 16, 32, S) == 0
    assert lib.mmf_glu_fwd(None, None, None, None, None, 4, 16, 0, S) == 0
    assert lib.mmf_glu_pack(None, None, 0, 16, None, S) == 0
    assert lib.mmf_ternary_gemm_glu(A, B, C, D, E, A, 4, 16, 24, S) == 2
    assert lib.mmf_ternary_gemm_glu(A, B, None, D, E, A, 4, 16, 32, S) == 1
    assert lib.mmf_ternary_gemm_glu(A, B, C, D, E, BAD, 4, 16, 32, S) == 3


def test_bias_argument_checks(mmf):
    lib = _c(mmf)
    assert lib.mmf_bitlinear_fwd_bias(A, 0, B, C, D, E, A, 4, 16, 6, S) == 2    # N % 4
    assert lib.mmf_bitlinear_fwd_bias(A, 0, B, C, D, None, A, 4, 16, 8, S) == 1
    assert lib.mmf_bitlinear_fwd_bias(A, 0, B, C, D, BAD, A, 4, 16, 8, S) == 3
    assert lib.mmf_bitlinear_fwd_bias(A, 2, B, C, D, E, A, 4, 16, 8, S) == 4
    assert lib.mmf_bitlinear_fwd_bias(A, 0, B, C, D, E, A, 4, 24, 8, S) == 2
    assert lib.mmf_bitlinear_fwd_bias(None, 0, None, None, None, None, None, 0, 16, 8, S) == 0


def test_mlgru_argument_checks(mmf):
    lib = _c(mmf)
    W = 0x100000   # aligned stand-in workspace
    # projection: d a positive multiple of 16, K as for the forward
    for d in (0, -16, 24):
        assert lib.mmf_mlgru_proj(A, 0, B, C, D, E, A, B, 4, 16, d, None, 0, S) == 2
    assert lib.mmf_mlgru_proj(A, 0, B, C, D, E, A, B, 4, 24, 16, None, 0, S) == 2
    assert lib.mmf_mlgru_proj(None, 0, B, C, D, E, A, B, 4, 16, 16, None, 0, S) == 1
    assert lib.mmf_mlgru_proj(A, 0, B, None, D, E, A, B, 4, 16, 16, None, 0, S) == 1
    assert lib.mmf_mlgru_proj(A, 0, B, C, None, E, A, B, 4, 16, 16, None, 0, S) == 1
    assert lib.mmf_mlgru_proj(A, 0, B, C, D, E, A, None, 4, 16, 16, None, 0, S) == 1
    assert lib.mmf_mlgru_proj(A, 0, B, C, D, BAD, A, B, 4, 16, 16, None, 0, S) == 3
    assert lib.mmf_mlgru_proj(A, 0, B, C, D, E, BAD, B, 4, 16, 16, None, 0, S) == 3
    assert lib.mmf_mlgru_proj(A, 5, B, C, D, E, A, B, 4, 16, 16, None, 0, S) == 4
    need = mmf.mmf_mlgru_proj_workspace_bytes(4, 16, 16)
    assert need > 0 and need % 256 == 0
    assert lib.mmf_mlgru_proj(A, 0, B, C, D, E, A, B, 4, 16, 16, W, need - 1, S) == 6
    assert lib.mmf_mlgru_proj(A, 0, B, C, D, E, A, B, 4, 16, 16, W + 16, need, S) == 6
    assert lib.mmf_mlgru_proj(None, 0, None, None, None, None, None, None, 0, 16, 16, None, 0, S) == 0
    assert lib.mmf_mlgru_proj_q(A, B, C, D, E, A, B, C, 4, 16, 24, S) == 2
    assert lib.mmf_mlgru_proj_q(A, B, None, D, E, A, B, C, 4, 16, 16, S) == 1
    assert lib.mmf_mlgru_proj_q(A, B, C, D, E, BAD, B, C, 4, 16, 16, S) == 3
    assert lib.mmf_mlgru_proj_q(None, None, None, None, None, None, None, None, 0, 16, 16, S) == 0
    # recurrence
    assert lib.mmf_mlgru_scan(A, B, C, D, 2, 3, 24, None, 0, S) == 2
    assert lib.mmf_mlgru_scan(A, B, C, D, -1, 3, 16, None, 0, S) == 2
    assert lib.mmf_mlgru_scan(A, B, C, D, 2 ** 20, 2 ** 12, 16, None, 0, S) == 2   # B*T > 2^31-1
    assert lib.mmf_mlgru_scan(None, B, C, D, 2, 3, 16, None, 0, S) == 1
    assert lib.mmf_mlgru_scan(A, B, None, D, 2, 3, 16, None, 0, S) == 1
    assert lib.mmf_mlgru_scan(A, BAD, C, D, 2, 3, 16, None, 0, S) == 3
    assert lib.mmf_mlgru_scan(A, B, C, BAD, 2, 3, 16, None, 0, S) == 3
    assert lib.mmf_mlgru_scan(None, None, None, None, 0, 3, 16, None, 0, S) == 0
    assert lib.mmf_mlgru_scan(None, None, None, None, 2, 0, 16, None, 0, S) == 0
    # a short sequence is one chunk and needs no workspace; a long one does
    assert mmf.mmf_mlgru_scan_workspace_bytes(1, 1, 2048) == 0
    assert mmf.mmf_mlgru_scan_workspace_bytes(4, 16, 64) == 0
    need = mmf.mmf_mlgru_scan_workspace_bytes(1, 2048, 2048)
    assert need >= 3 * 2048 * 4 * 2 and need % 256 == 0
    assert lib.mmf_mlgru_scan(A, B, C, D, 1, 2048, 2048, W, need - 1, S) == 6
    # whole mixer
    assert lib.mmf_mlgru_fwd(A, 0, B, C, D, E, A, B, C, D, E, A, B, C, 1, 2, 24, None, 0, S) == 2
    assert lib.mmf_mlgru_fwd(A, 0, B, C, D, E, A, B, C, D, None, A, B, C, 1, 2, 32, None, 0, S) == 1
    assert lib.mmf_mlgru_fwd(A, 0, B, C, D, E, A, B, C, D, E, None, B, C, 1, 2, 32, None, 0, S) == 1
    assert lib.mmf_mlgru_fwd(A, 0, B, C, D, E, A, B, C, D, E, A, B, None, 1, 2, 32, None, 0, S) == 1
    assert lib.mmf_mlgru_fwd(A, 0, B, C, D, E, A, BAD, C, D, E, A, B, C, 1, 2, 32, None, 0, S) == 3
    assert lib.mmf_mlgru_fwd(A, 0, B, C, D, E, A, B, C, D, E, A, BAD, C, 1, 2, 32, None, 0, S) == 3
    assert lib.mmf_mlgru_fwd(A, 9, B, C, D, E, A, B, C, D, E, A, B, C, 1, 2, 32, None, 0, S) == 4
    need = mmf.mmf_mlgru_workspace_bytes(1, 2, 32)
    assert need >= 2 * 32 * 16 and need % 256 == 0
    assert lib.mmf_mlgru_fwd(A, 0, B, C, D, E, A, B, C, D, E, A, B, C, 1, 2, 32, W, need - 1, S) == 6
    assert lib.mmf_mlgru_fwd(None, 0, None, None, None, None, None, None, None, None, None, None,
                             None, None, 0, 2, 32, None, 0, S) == 0
    assert mmf.mmf_mlgru_workspace_bytes(1, 2048, 2048) >= 2048 * 2048 * 16


def test_train_and_bwd_argument_checks(mmf):
    lib = _c(mmf)
    W = 0x100000
    # training forward: shape, GEMM limits, bias needs N % 4 == 0
    assert lib.mmf_bitlinear_train_fwd(A, 0, B, C, D, E, A, B, C, D, E, 4, 24, 8, None, 0, S) == 2
    assert lib.mmf_bitlinear_train_fwd(A, 0, B, C, D, E, A, B, C, D, E, 4, 16, 2 ** 24 + 4, None, 0, S) == 2
    assert lib.mmf_bitlinear_train_fwd(A, 0, B, C, D, E, A, B, C, D, E, 4, 16, 6, None, 0, S) == 2
    assert lib.mmf_bitlinear_train_fwd(A, 0, B, None, None, E, A, B, C, D, E, 4, 16, 6, None, 0, S) == 1
    assert lib.mmf_bitlinear_train_fwd(A, 0, B, None, None, E, A, B, C, D, E, 4, 16, 8, None, 0, S) == 1
    assert lib.mmf_bitlinear_train_fwd(A, 0, B, C, None, E, A, B, None, D, E, 4, 16, 8, None, 0, S) == 1
    assert lib.mmf_bitlinear_train_fwd(A, 0, B, C, None, E, A, B, C, D, BAD, 4, 16, 8, None, 0, S) == 3
    assert lib.mmf_bitlinear_train_fwd(A, 7, B, C, None, E, A, B, C, D, E, 4, 16, 8, None, 0, S) == 4
    need = mmf.mmf_bitlinear_train_workspace_bytes(4, 16, 8)
    assert need > 0 and need % 256 == 0
    assert lib.mmf_bitlinear_train_fwd(A, 0, B, C, None, E, A, B, C, D, E, 4, 16, 8, W, need - 1, S) == 6
    assert lib.mmf_bitlinear_train_fwd(None, 0, None, None, None, None, None, None, None, None, None,
                                       0, 16, 8, None, 0, S) == 0
    # backward
    assert lib.mmf_bitlinear_bwd(A, B, 0, C, D, E, A, B, C, D, E, A, B, 4, 24, 8, None, 0, S) == 2
    assert lib.mmf_bitlinear_bwd(None, B, 0, C, D, E, A, B, C, D, E, A, B, 4, 16, 8, None, 0, S) == 1
    assert lib.mmf_bitlinear_bwd(A, B, 0, C, None, E, A, B, C, D, E, A, B, 4, 16, 8, None, 0, S) == 1
    assert lib.mmf_bitlinear_bwd(A, B, 0, C, D, E, A, B, C, D, None, A, B, 4, 16, 8, None, 0, S) == 1
    assert lib.mmf_bitlinear_bwd(A, B, 0, C, D, E, A, B, C, D, E, BAD, B, 4, 16, 8, None, 0, S) == 3
    assert lib.mmf_bitlinear_bwd(A, B, 2, C, D, E, A, B, C, D, E, A, B, 4, 16, 8, None, 0, S) == 4
    need = mmf.mmf_bitlinear_bwd_workspace_bytes(4, 16, 8)
    assert need >= 16 * 8 * 2 + 4 * 16 * 6 and need % 256 == 0
    assert lib.mmf_bitlinear_bwd(A, B, 0, C, D, E, A, B, C, D, E, A, B, 4, 16, 8, W, need - 1, S) == 6
    assert lib.mmf_bitlinear_bwd(None, None, 0, None, None, None, None, None, None, None, None, None,
                                 None, 0, 16, 8, None, 0, S) == 0


def test_status_codes_follow_the_boundary():
    """The numbering the boundary fixes: OK 0, NULL 1, SHAPE 2, ALIGN 3,
    DTYPE 4, HIP 5 (then this library's WORKSPACE 6 and ARG 7)."""
    text = open(HEADER).read()
    codes = dict(re.findall(r"#define (MMF_[A-Z_0-9]+) (-?\d+)", text))
    want = {"MMF_OK": "0", "MMF_ERR_NULL": "1", "MMF_ERR_SHAPE": "2", "MMF_ERR_ALIGN": "3",
            "MMF_ERR_DTYPE": "4", "MMF_ERR_HIP": "5", "MMF_ERR_WORKSPACE": "6", "MMF_ERR_ARG": "7"}
    for k, v in want.items():
        assert codes.get(k) == v, (k, codes.get(k))


def test_boundary_signatures():
    """The three calls of the boundary keep their argument lists:
    mmf_ternarize_weights(W, N, K, Wpacked, w_scale, stream),
    mmf_bitlinear_fwd(x, gamma, Wpacked, w_scale, y, M, K, N, stream),
    mmf_act_quant(x, gamma, q, a_scale, M, K, stream)."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)

    def params(name):
        m = re.search(r"\b" + name + r"\s*\(([^)]*)\)", text)
        assert m, name
        return [re.findall(r"(\w+)\s*$", p.strip())[0] for p in m.group(1).split(",")]

    assert params("mmf_ternarize_weights") == ["W", "N", "K", "Wpacked", "w_scale", "stream"]
    assert params("mmf_bitlinear_fwd") == ["x", "gamma", "Wpacked", "w_scale", "y", "M", "K", "N",
                                           "stream"]
    assert params("mmf_act_quant") == ["x", "gamma", "q", "a_scale", "M", "K", "stream"]
    assert params("mmf_act_quant_f32") == ["x", "gamma", "q", "a_scale", "M", "K", "stream"]
    assert params("mmf_ternary_gemm_i32") == ["q", "Wpacked", "acc", "M", "K", "N", "stream"]


def test_shapes_past_the_kernel_offsets_are_rejected_up_front(mmf):
    """Shapes the contraction kernel cannot address with its 32-bit offsets
    return MMF_ERR_SHAPE from the host checks, before anything is enqueued
    (the stand-in pointers are never dereferenced, so reaching a launch would
    fault the test process instead)."""
    lib = _c(mmf)
    W = 0x100000
    big_n = 1 << 21            # M = 65 takes the MFMA kernel: output row slices < 256 rows
    huge = (1 << 27) + 16      # packed weights (K/16) * N * 4 >= 2^31 at K = 256
    for M, K, N in ((65, 16, big_n), (4096, 256, huge), (65, 16, (1 << 24) + 4)):
        assert lib.mmf_bitlinear_fwd(A, B, C, D, E, M, K, N, S) == 2
        assert lib.mmf_bitlinear_fwd_f32(A, B, C, D, E, M, K, N, S) == 2
        assert lib.mmf_bitlinear_fwd_ws(A, 0, B, C, D, E, M, K, N, W, 1 << 40, S) == 2
        assert lib.mmf_ternary_gemm_dequant(A, B, C, D, E, A, M, K, N, S) == 2
        assert lib.mmf_ternary_gemm_i32(A, B, C, M, K, N, S) == 2
        assert lib.mmf_bitlinear_fwd_bias(A, 0, B, C, D, E, A, M, K, N, S) == 2
        assert lib.mmf_bitlinear_train_fwd(A, 0, B, C, None, E, A, B, C, D, E, M, K, N, None, 0, S) == 2
        assert lib.mmf_glu_fwd(A, B, C, D, E, M, K, N // 2, S) == 2
        assert lib.mmf_ternary_gemm_glu(A, B, C, D, E, A, M, K, N // 2, S) == 2
    # the MLGRU projection: 3d columns past the MFMA kernel's slice limit
    d = 1 << 20
    assert lib.mmf_mlgru_proj(A, 0, B, C, D, E, A, B, 65, 16, d, None, 0, S) == 2
    assert lib.mmf_mlgru_proj_q(A, B, C, D, E, A, B, C, 65, 16, d, S) == 2


def test_backward_shapes_past_its_offsets_are_rejected_up_front(mmf):
    """The backward's 32-bit offsets: dW [N][K] of 2^31 bytes or more, the
    re-packed codes, and dO rows too long for a 128-row slice return
    MMF_ERR_SHAPE (and a zero workspace size) before anything is enqueued."""
    lib = _c(mmf)
    for M, K, N in ((64, 2048, 1 << 18), (64, 1 << 16, 1 << 15), (64, 16, (1 << 23) + 8)):
        assert lib.mmf_bitlinear_bwd_workspace_bytes(M, K, N) == 0
        assert lib.mmf_bitlinear_bwd(A, B, 0, None, C, D, E, A, B, C, D, None, None, M, K, N, None, 0, S) == 2
    # just inside: dW of 2^31 - 2^13 bytes
    assert lib.mmf_bitlinear_bwd_workspace_bytes(64, 2048, (1 << 18) - 1) > 0


def test_noalloc_argument_checks(mmf):
    """The forward without allocation: the same checks as the forward, and
    scratch needs past its static array rejected before anything is
    enqueued."""
    lib = _c(mmf)
    assert mmf.mmf_bitlinear_noalloc_max_bytes() == 64 << 20
    assert lib.mmf_bitlinear_fwd_noalloc(A, 0, B, C, D, E, 4, 24, 8, S) == 2
    assert lib.mmf_bitlinear_fwd_noalloc(A, 2, B, C, D, E, 4, 16, 8, S) == 4
    assert lib.mmf_bitlinear_fwd_noalloc(None, 0, B, C, D, E, 4, 16, 8, S) == 1
    assert lib.mmf_bitlinear_fwd_noalloc(A, 0, B, C, BAD, E, 4, 16, 8, S) == 1 or \
        lib.mmf_bitlinear_fwd_noalloc(A, 0, B, C, D, BAD, 4, 16, 8, S) == 3
    assert lib.mmf_bitlinear_fwd_noalloc(A, 0, B, C, D, BAD, 4, 16, 8, S) == 3
    assert lib.mmf_bitlinear_fwd_noalloc(None, 0, None, None, None, None, 0, 16, 8, S) == 0
    # 65536 tokens of 1040 features: 68 MB of q, past the 64 MiB array
    assert lib.mmf_bitlinear_fwd_noalloc(A, 0, B, C, D, E, 65536, 1040, 64, S) == 6
    assert lib.mmf_bitlinear_fwd_noalloc(A, 0, B, C, D, E, 65, 16, 1 << 21, S) == 2


def test_prefill_tile_plan(mmf):
    """The planner's choice on 256 compute units (host only): the parity shapes
    take the kernel forms their tests name, and the workloads theirs."""
    P = mmf.mmf_prefill_tile_plan
    glu, affine, raw = mmf.MMF_EPILOGUE_GLU, mmf.MMF_EPILOGUE_AFFINE, mmf.MMF_EPILOGUE_RAW_I32
    # tests/test_gpu_parity.py and tests/test_gpu_glu.py
    assert P(300, 1040, 2000) == "64x256"
    assert P(1000, 336, 6000) == "64x512"
    assert P(1100, 528, 8000) == "128x512"              # one round of 144 wide tiles
    assert P(3000, 400, 8200) == "128x256_paired"       # 408 wide tiles
    assert P(3000, 400, 8200, raw) == "128x256_paired"
    assert P(3000, 400, 2 * 4112, glu) == "128x256_paired"
    assert P(37, 272, 300 + 2) == "256x256"             # N % 4 != 0
    # workloads
    assert P(16384, 5120, 27648) == "128x512"           # large: K > 4096
    assert P(8192, 2048, 11264) == "128x256_paired"     # glu_up
    assert P(8192, 2048, 11264, glu) == "128x256_paired"  # glu_gate
    assert P(8192, 5632, 2048) == "128x512"             # glu_down: K > 4096
    assert P(2048, 2048, 6144, affine) == "128x512"     # MLGRU gate projection: affine epilogue
    assert P(2048, 2048, 2048) == "64x256"              # MLGRU output projection
    assert P(16384, 1024, 1024) == "128x256_paired"     # training forward at d = 1024: a full round, K <= 2048
    # a single round at K = 3072 keeps the wide tile; two rounds take the pairs
    assert P(2048, 3072, 8192) == "128x512"
    assert P(4096, 3072, 8192) == "128x256_paired"
    # invalid arguments
    for args in ((0, 16, 16, 0, 256), (16, 15, 16, 0, 256), (16, 16, 0, 0, 256), (16, 16, 16, 0, 0),
                 (16, 16, 48, glu, 256)):
        with pytest.raises(mmf.MMFError, match="MMF_ERR_SHAPE"):
            P(*args)
    with pytest.raises(mmf.MMFError):
        P(16, 16, 16, 9, 256)
