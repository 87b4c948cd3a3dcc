"""The forward that allocates nothing (mmf_bitlinear_fwd_noalloc), called
through the C ABI: its output must equal mmf_bitlinear_fwd_ws's bit for bit
(the same kernels, with the scratch in the library's static device array
instead of caller memory) and meet the parity bar against the oracle.  Two
calls in a row on the shared array, the second with a smaller input; then a
decode-sized call (no scratch) and a float32-activation call."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import workloads
from _parity import compare_q, compare_y, dev, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mmf():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2406_02528_amd as m
    return m


def _case(seed, M, K, N, f32=False):
    rs = np.random.default_rng(seed)
    bits, xf, g, W = workloads.random_case(rs, M, K, N)
    if f32:
        x = torch.from_numpy(xf).to(dev())
    else:
        x = torch.from_numpy(bits.view(np.int16)).to(dev()).view(torch.bfloat16)
    return x, xf, g, W


def _noalloc(mmf, x, g_d, Wp, ws, y):
    M, K = x.shape
    N = Wp.shape[1]
    st = mmf._lib.mmf_bitlinear_fwd_noalloc(
        ctypes.c_void_p(x.data_ptr()), int(x.dtype == torch.float32), ctypes.c_void_p(g_d.data_ptr()),
        ctypes.c_void_p(Wp.data_ptr()), ctypes.c_void_p(ws.data_ptr()), ctypes.c_void_p(y.data_ptr()),
        M, K, N, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0, mmf.mmf_status_string(st)


def _check(mmf, seed, M, K, N, f32=False):
    log(f"[no_alloc] seed={seed} M={M} K={K} N={N} f32={f32}")
    x, xf, g, W = _case(seed, M, K, N, f32)
    g_d = torch.from_numpy(g).to(dev())
    Wp, ws = mmf.ternarize(torch.from_numpy(W).to(dev()))
    y_na = torch.full((M, N), float("nan"), dtype=torch.float32, device=dev())
    _noalloc(mmf, x, g_d, Wp, ws, y_na)
    y_ws = torch.full((M, N), float("nan"), dtype=torch.float32, device=dev())
    wsb = torch.empty(max(1, mmf.mmf_bitlinear_workspace_bytes(M, K)), dtype=torch.uint8, device=dev())
    mmf.mmf_bitlinear_fwd_ws(x, g_d, Wp, ws, y_ws, wsb)
    torch.cuda.synchronize()
    a, b = y_na.cpu().numpy(), y_ws.cpu().numpy()
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), "differs from mmf_bitlinear_fwd_ws"
    # the parity bar against the oracle
    t, ws_ref = oracle.weight_quant(W)
    q_ref, a_ref = oracle.rmsnorm_act_quant(xf, g)
    acc = oracle.ternary_accumulate(q_ref, t)
    y_ref = oracle.dequant(acc, a_ref, ws_ref)
    q_gpu = torch.empty((M, K), dtype=torch.int8, device=dev())
    a_gpu = torch.empty((M,), dtype=torch.float32, device=dev())
    mmf.mmf_act_quant(x, g_d, q_gpu, a_gpu)
    torch.cuda.synchronize()
    flips, _ = compare_q(q_gpu.cpu().numpy(), q_ref)
    mask = np.zeros(M, bool)
    mask[flips] = True
    compare_y(a, y_ref, acc, mask)


def test_noalloc_two_calls_then_smaller(mmf):
    assert mmf.mmf_bitlinear_noalloc_max_bytes() == 64 << 20
    # prefill shapes (the scratch is used): a larger call, then a smaller one
    # on the same array
    _check(mmf, 11, 300, 2064, 1040)
    _check(mmf, 12, 97, 512, 264)


def test_noalloc_decode_and_f32(mmf):
    _check(mmf, 13, 5, 2048, 640)            # fused decode launches, no scratch
    _check(mmf, 14, 129, 256, 520, f32=True)


def test_noalloc_rejects_past_its_array(mmf):
    # M*K + 8M past 64 MiB: rejected on the host before anything is enqueued
    x = torch.zeros((65536, 1040), dtype=torch.bfloat16, device=dev())
    Wp = torch.zeros((1040 // 16, 64), dtype=torch.int32, device=dev())
    ws = torch.ones((1,), dtype=torch.float32, device=dev())
    y = torch.full((65536, 64), 7.0, dtype=torch.float32, device=dev())
    st = mmf._lib.mmf_bitlinear_fwd_noalloc(
        ctypes.c_void_p(x.data_ptr()), 0, None, ctypes.c_void_p(Wp.data_ptr()),
        ctypes.c_void_p(ws.data_ptr()), ctypes.c_void_p(y.data_ptr()), 65536, 1040, 64,
        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 6   # MMF_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert bool((y == 7.0).all()), "output touched after a rejected call"
