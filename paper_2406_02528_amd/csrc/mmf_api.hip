// C ABI of the fused BitLinear library: argument checks on the host, scratch
// management and kernel dispatch.  Nothing is enqueued before every argument
// has been checked.
#include <atomic>
#include <cstdint>
#include <cstring>
#include <mutex>

#include "mmf.h"
#include "mmf_launch.h"

namespace {

constexpr int64_t kMaxK = int64_t(1) << 20;
constexpr int64_t kMaxMN = 0x7FFFFFFF;
constexpr int kDecodeMaxTokens = mmf::kDecodeMaxTokens;
constexpr size_t kScratchAlign = 256;

std::atomic<int> g_path{MMF_PATH_AUTO};

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Shape rules shared by every entry point that takes K.
int check_shape(int64_t M, int64_t K, int64_t N) {
  if (K <= 0 || K > kMaxK || (K % 16) != 0) return MMF_ERR_SHAPE;
  if (M < 0 || M > kMaxMN || N < 0 || N > kMaxMN) return MMF_ERR_SHAPE;
  return MMF_OK;
}

int hip_status(hipError_t e) { return e == hipSuccess ? MMF_OK : MMF_ERR_HIP; }

// Layout of the forward's scratch: q [M][K] int8, a_scale [M] f32, rowsum [M] i32.
struct FwdScratch {
  size_t q_off, a_off, r_off, total;
};
FwdScratch fwd_scratch(int64_t M, int64_t K) {
  FwdScratch s;
  s.q_off = 0;
  s.a_off = round_up(static_cast<size_t>(M) * static_cast<size_t>(K), kScratchAlign);
  s.r_off = s.a_off + round_up(static_cast<size_t>(M) * 4, kScratchAlign);
  s.total = s.r_off + round_up(static_cast<size_t>(M) * 4, kScratchAlign);
  return s;
}

// Automatic choice: up to decode_max_tokens(K) tokens run as decode launches
// of at most 16 tokens each, when the decode kernel takes such a slice (its
// LDS holds q of 16 tokens up to K = 7680); more go to the MFMA kernel, whose
// time at a small M is one tile's k loop (latency-bound, ~0.6-0.9 us per 128
// of K).  Measured forward calls from x, decode slices at 16 / 32 / 48 / 64
// tokens against the MFMA kernel at 16-128 tokens: K = 1024, N = 4096: 5.0 /
// 9.5 / 13.9 / 18.1 us against 10.2-11.8; K = 2048, N = 6144: 6.7 / 12.7 /
// 18.6 / 24.5 against 15.2-17.2; K = 4096, N = 11008: 9.2 / 14.1 / 18.8 /
// 23.6 against 24.0-26.4; K = 5120, N = 15360: 11.5 / 16.7 / 21.6 / 26.8
// against 35.2-37.3.  So 32 tokens at K <= 2048, 64 beyond.  MMF_PATH_GEMV
// forces the decode kernels for every M (slices they cannot hold then go to
// the gemv kernel, which reads q from global memory); MMF_PATH_GEMM forces
// the MFMA kernel.
int64_t decode_max_tokens(int64_t K) { return K <= 2048 ? 32 : 64; }
bool use_decode(int64_t M, int64_t K, int64_t N, bool from_x, bool x_is_f32) {
  const int p = g_path.load(std::memory_order_relaxed);
  if (p == MMF_PATH_GEMV) return true;
  if (p == MMF_PATH_GEMM) return false;
  if (M > decode_max_tokens(K)) return false;
  return mmf::decode_fits(M < kDecodeMaxTokens ? M : kDecodeMaxTokens, static_cast<int>(K), N, from_x,
                          x_is_f32);
}

// Contraction from quantised activations.  Decode-sized slices of at most 16
// tokens keep q in LDS when it fits, else read it from global memory.
hipError_t contract(const mmf::ContractArgs& a, hipStream_t stream) {
  if (!use_decode(a.M, a.K, a.N, false, false)) return mmf::launch_gemm(a, stream);
  for (int64_t m0 = 0; m0 < a.M; m0 += kDecodeMaxTokens) {
    const int64_t mt = a.M - m0 < kDecodeMaxTokens ? a.M - m0 : kDecodeMaxTokens;
    const bool raw = a.epilogue == mmf::Epilogue::kRawI32;
    void* out = raw ? static_cast<void*>(static_cast<int32_t*>(a.out) + m0 * a.N)
                    : static_cast<void*>(static_cast<float*>(a.out) + m0 * a.N);
    const float* as = a.a_scale ? a.a_scale + m0 : nullptr;
    hipError_t e;
    if (mmf::decode_fits(mt, a.K, a.N, false, false)) {
      mmf::DecodeArgs d{nullptr, false, nullptr, a.q + m0 * a.K, as, a.q_rowsum + m0,
                        a.Wpacked, a.w_scale, out, mt, a.K, a.N, a.epilogue};
      e = mmf::launch_decode(d, stream);
    } else {
      mmf::ContractArgs s{a.q + m0 * a.K, as, a.q_rowsum + m0, a.Wpacked, a.w_scale, out,
                          mt, a.K, a.N, a.epilogue};
      e = mmf::launch_gemv(s, stream);
    }
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// The whole forward runs as fused decode launches (no scratch) when every
// slice of at most 16 tokens fits the fused kernel.
bool fused_decode(int64_t M, int64_t K, int64_t N, bool x_is_f32) {
  if (!use_decode(M, K, N, true, x_is_f32)) return false;
  const int64_t mt = M < kDecodeMaxTokens ? M : kDecodeMaxTokens;
  return mmf::decode_fits(mt, static_cast<int>(K), N, true, x_is_f32);
}

// Shape limits of the kernels a call will run, checked before anything is
// enqueued (MMF_ERR_SHAPE).  check_contract: the contraction from quantised
// activations (contract() above); check_gemm: the MFMA kernel alone;
// check_from_x: a forward from x, which runs fused decode launches when they
// fit and otherwise act-quant followed by `gemm_only ? the MFMA kernel :
// contract()`.
int check_gemm(int64_t K, int64_t N) {
  return mmf::gemm_row_slice(K, N) > 0 ? MMF_OK : MMF_ERR_SHAPE;
}
int check_contract(int64_t M, int64_t K, int64_t N) {
  if (M == 0 || N == 0 || use_decode(M, K, N, false, false)) return MMF_OK;
  return check_gemm(K, N);
}
int check_from_x(int64_t M, int64_t K, int64_t N, bool x_is_f32, bool gemm_only) {
  if (M == 0 || N == 0 || fused_decode(M, K, N, x_is_f32)) return MMF_OK;
  return gemm_only ? check_gemm(K, N) : check_contract(M, K, N);
}
int check_dtype(int x_is_f32) { return (x_is_f32 == 0 || x_is_f32 == 1) ? MMF_OK : MMF_ERR_DTYPE; }

hipError_t run_fused_decode(const void* x, bool x_is_f32, const float* gamma,
                            const uint32_t* Wpacked, const float* w_scale, float* y, int64_t M,
                            int64_t K, int64_t N, hipStream_t stream) {
  const size_t xsz = x_is_f32 ? 4 : 2;
  for (int64_t m0 = 0; m0 < M; m0 += kDecodeMaxTokens) {
    const int64_t mt = M - m0 < kDecodeMaxTokens ? M - m0 : kDecodeMaxTokens;
    mmf::DecodeArgs d{static_cast<const char*>(x) + m0 * K * xsz, x_is_f32, gamma, nullptr,
                      nullptr, nullptr, Wpacked, w_scale, y + m0 * N, mt,
                      static_cast<int>(K), N, mmf::Epilogue::kDequantF32};
    const hipError_t e = mmf::launch_decode(d, stream);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Checks of the forward's arguments shared by the allocating and _ws forms.
int check_fwd(const void* x, bool x_is_f32, const float* gamma, const uint32_t* Wpacked,
              const float* w_scale, const float* y, int64_t M, int64_t K, int64_t N,
              bool gemm_only = false) {
  if (int st = check_shape(M, K, N)) return st;
  if (M == 0 || N == 0) return MMF_OK;
  if (int st = check_from_x(M, K, N, x_is_f32, gemm_only)) return st;
  if (!x || !Wpacked || !w_scale || !y) return MMF_ERR_NULL;
  if (!aligned16(x) || !aligned16(Wpacked) || !aligned16(y) || (gamma && !aligned16(gamma)))
    return MMF_ERR_ALIGN;
  return MMF_OK;
}

int run_fwd(const void* x, bool x_is_f32, const float* gamma, const uint32_t* Wpacked,
            const float* w_scale, float* y, int64_t M, int64_t K, int64_t N, char* scratch,
            hipStream_t stream) {
  if (fused_decode(M, K, N, x_is_f32))
    return hip_status(run_fused_decode(x, x_is_f32, gamma, Wpacked, w_scale, y, M, K, N, stream));
  const FwdScratch s = fwd_scratch(M, K);
  int8_t* q = reinterpret_cast<int8_t*>(scratch + s.q_off);
  float* a_scale = reinterpret_cast<float*>(scratch + s.a_off);
  int32_t* rowsum = reinterpret_cast<int32_t*>(scratch + s.r_off);
  hipError_t e = mmf::launch_act_quant(x, x_is_f32, gamma, q, a_scale, rowsum, M,
                                       static_cast<int>(K), stream);
  if (e != hipSuccess) return MMF_ERR_HIP;
  mmf::ContractArgs a{q, a_scale, rowsum, Wpacked, w_scale, y, M, static_cast<int>(K), N,
                      mmf::Epilogue::kDequantF32};
  return hip_status(contract(a, stream));
}

int fwd_alloc(const void* x, bool x_is_f32, const float* gamma, const uint32_t* Wpacked,
              const float* w_scale, float* y, int64_t M, int64_t K, int64_t N,
              hipStream_t stream) {
  if (int st = check_fwd(x, x_is_f32, gamma, Wpacked, w_scale, y, M, K, N)) return st;
  if (M == 0 || N == 0) return MMF_OK;
  if (fused_decode(M, K, N, x_is_f32))
    return hip_status(run_fused_decode(x, x_is_f32, gamma, Wpacked, w_scale, y, M, K, N, stream));
  const FwdScratch s = fwd_scratch(M, K);
  void* scratch = nullptr;
  if (hipMallocAsync(&scratch, s.total, stream) != hipSuccess) return MMF_ERR_HIP;
  const int st = run_fwd(x, x_is_f32, gamma, Wpacked, w_scale, y, M, K, N,
                         static_cast<char*>(scratch), stream);
  const hipError_t fe = hipFreeAsync(scratch, stream);
  if (st != MMF_OK) return st;
  return hip_status(fe);
}

int act_quant_common(const void* x, int x_is_f32, const float* gamma, int8_t* q,
                     float* a_scale, int32_t* q_rowsum, int64_t M, int64_t K,
                     hipStream_t stream) {
  if (int st = check_dtype(x_is_f32)) return st;
  if (int st = check_shape(M, K, 0)) return st;
  if (M == 0) return MMF_OK;
  if (!x || !q || !a_scale) return MMF_ERR_NULL;
  if (!aligned16(x) || !aligned16(q) || !aligned16(a_scale) || (gamma && !aligned16(gamma)) ||
      (q_rowsum && !aligned16(q_rowsum)))
    return MMF_ERR_ALIGN;
  return hip_status(mmf::launch_act_quant(x, x_is_f32 == 1, gamma, q, a_scale, q_rowsum, M,
                                          static_cast<int>(K), stream));
}

// Runs `run(scratch)` on the caller's workspace (checked against `need`), or
// on stream-ordered scratch allocated here when `workspace` is NULL.
template <class F>
int with_workspace(void* workspace, size_t workspace_bytes, size_t need, hipStream_t stream, F&& run) {
  if (workspace != nullptr) {
    if ((reinterpret_cast<uintptr_t>(workspace) & (kScratchAlign - 1)) != 0 || workspace_bytes < need)
      return MMF_ERR_WORKSPACE;
    return run(static_cast<char*>(workspace));
  }
  if (need == 0) return run(nullptr);
  void* p = nullptr;
  if (hipMallocAsync(&p, need, stream) != hipSuccess) return MMF_ERR_HIP;
  const int st = run(static_cast<char*>(p));
  const hipError_t fe = hipFreeAsync(p, stream);
  if (st != MMF_OK) return st;
  return hip_status(fe);
}

// GLU (gated up-projection): x -> RMSNorm + quantisation -> the interleaved
// gate/up contraction with the SiLU(g) * u epilogue: fused decode launches for
// the token counts the decode kernel takes, the MFMA kernel otherwise.
int check_glu(const void* x, bool x_is_f32, const float* gamma, const uint32_t* Wgu,
              const float* w_scales, const float* p, int64_t M, int64_t K, int64_t L) {
  if (L < 0 || L > kMaxMN / 2 || (L % 16) != 0) return MMF_ERR_SHAPE;
  if (int st = check_shape(M, K, 2 * L)) return st;
  if (M == 0 || L == 0) return MMF_OK;
  if (int st = check_from_x(M, K, 2 * L, x_is_f32, true)) return st;
  if (!x || !Wgu || !w_scales || !p) return MMF_ERR_NULL;
  if (!aligned16(x) || !aligned16(Wgu) || !aligned16(p) || (gamma && !aligned16(gamma)))
    return MMF_ERR_ALIGN;
  return MMF_OK;
}

int run_glu(const void* x, bool x_is_f32, const float* gamma, const uint32_t* Wgu,
            const float* w_scales, float* p, int64_t M, int64_t K, int64_t L, char* scratch,
            hipStream_t stream) {
  // few tokens: fused decode launches with the GLU epilogue (no scratch)
  if (fused_decode(M, K, 2 * L, x_is_f32)) {
    const size_t xsz = x_is_f32 ? 4 : 2;
    for (int64_t m0 = 0; m0 < M; m0 += kDecodeMaxTokens) {
      const int64_t mt = M - m0 < kDecodeMaxTokens ? M - m0 : kDecodeMaxTokens;
      mmf::DecodeArgs d{static_cast<const char*>(x) + m0 * K * xsz, x_is_f32, gamma, nullptr,
                        nullptr, nullptr, Wgu, w_scales, p + m0 * L, mt,
                        static_cast<int>(K), 2 * L, mmf::Epilogue::kGluF32};
      if (mmf::launch_decode(d, stream) != hipSuccess) return MMF_ERR_HIP;
    }
    return MMF_OK;
  }
  const FwdScratch s = fwd_scratch(M, K);
  int8_t* q = reinterpret_cast<int8_t*>(scratch + s.q_off);
  float* a_scale = reinterpret_cast<float*>(scratch + s.a_off);
  int32_t* rowsum = reinterpret_cast<int32_t*>(scratch + s.r_off);
  hipError_t e = mmf::launch_act_quant(x, x_is_f32, gamma, q, a_scale, rowsum, M,
                                       static_cast<int>(K), stream);
  if (e != hipSuccess) return MMF_ERR_HIP;
  mmf::ContractArgs a{q, a_scale, rowsum, Wgu, w_scales, p, M, static_cast<int>(K), 2 * L,
                      mmf::Epilogue::kGluF32};
  return hip_status(mmf::launch_gemm(a, stream));
}

int glu_alloc(const void* x, bool x_is_f32, const float* gamma, const uint32_t* Wgu,
              const float* w_scales, float* p, int64_t M, int64_t K, int64_t L,
              hipStream_t stream) {
  if (int st = check_glu(x, x_is_f32, gamma, Wgu, w_scales, p, M, K, L)) return st;
  if (M == 0 || L == 0) return MMF_OK;
  // the fused decode launches need no scratch
  const size_t need = fused_decode(M, K, 2 * L, x_is_f32) ? 0 : fwd_scratch(M, K).total;
  return with_workspace(nullptr, 0, need, stream, [&](char* scratch) {
    return run_glu(x, x_is_f32, gamma, Wgu, w_scales, p, M, K, L, scratch, stream);
  });
}

// ---- affine forward (bias and per-segment activations after the dequant) ----

// Fused decode launches when every slice of at most 16 tokens fits the fused
// kernel, else activation quantisation into `scratch` (fwd_scratch) and the
// MFMA kernel for every M.
int run_affine(const void* x, bool x_is_f32, const float* gamma, const uint32_t* Wpacked,
               const float* w_scales, const mmf::Affine& aff, float* y, int64_t M, int64_t K,
               int64_t N, char* scratch, hipStream_t stream) {
  if (fused_decode(M, K, N, x_is_f32)) {
    const size_t xsz = x_is_f32 ? 4 : 2;
    for (int64_t m0 = 0; m0 < M; m0 += kDecodeMaxTokens) {
      const int64_t mt = M - m0 < kDecodeMaxTokens ? M - m0 : kDecodeMaxTokens;
      mmf::DecodeArgs d{static_cast<const char*>(x) + m0 * K * xsz, x_is_f32, gamma, nullptr,
                        nullptr, nullptr, Wpacked, w_scales, y + m0 * N, mt,
                        static_cast<int>(K), N, mmf::Epilogue::kAffineF32, aff};
      if (mmf::launch_decode(d, stream) != hipSuccess) return MMF_ERR_HIP;
    }
    return MMF_OK;
  }
  const FwdScratch s = fwd_scratch(M, K);
  int8_t* q = reinterpret_cast<int8_t*>(scratch + s.q_off);
  float* a_scale = reinterpret_cast<float*>(scratch + s.a_off);
  int32_t* rowsum = reinterpret_cast<int32_t*>(scratch + s.r_off);
  if (mmf::launch_act_quant(x, x_is_f32, gamma, q, a_scale, rowsum, M, static_cast<int>(K), stream) !=
      hipSuccess)
    return MMF_ERR_HIP;
  mmf::ContractArgs a{q, a_scale, rowsum, Wpacked, w_scales, y, M, static_cast<int>(K), N,
                      mmf::Epilogue::kAffineF32, aff};
  return hip_status(mmf::launch_gemm(a, stream));
}

bool aligned16_or_null(const void* p) { return p == nullptr || aligned16(p); }

// ---- MLGRU ----
constexpr uint32_t kMlgruActs = mmf::kActSigmoidLb | (mmf::kActSilu << 2) | (mmf::kActIdentity << 4);

int check_mlgru_d(int64_t d) {
  if (d <= 0 || d % 16 != 0 || d > kMaxMN / 3) return MMF_ERR_SHAPE;
  return MMF_OK;
}

int check_mlgru_proj(const void* x, const float* gamma, const uint32_t* Wfcg, const float* w_scales,
                     const float* bias, const float* lb, const float* fcg, int64_t M, int64_t K,
                     int64_t d) {
  if (int st = check_mlgru_d(d)) return st;
  if (int st = check_shape(M, K, 3 * d)) return st;
  if (M == 0) return MMF_OK;
  if (!x || !Wfcg || !w_scales || !fcg) return MMF_ERR_NULL;
  if (!aligned16(x) || !aligned16(Wfcg) || !aligned16(fcg) || !aligned16_or_null(gamma) ||
      !aligned16_or_null(bias) || !aligned16_or_null(lb))
    return MMF_ERR_ALIGN;
  return MMF_OK;
}

int check_mlgru_scan(const float* fcg, const float* h0, const float* o, const float* h_last,
                     int64_t B, int64_t T, int64_t d) {
  if (int st = check_mlgru_d(d)) return st;
  if (B < 0 || T < 0 || B > kMaxMN || T > kMaxMN || (T > 0 && B > kMaxMN / T)) return MMF_ERR_SHAPE;
  if (B == 0 || T == 0) return MMF_OK;
  if (!fcg || !o) return MMF_ERR_NULL;
  if (!aligned16(fcg) || !aligned16(o) || !aligned16_or_null(h0) || !aligned16_or_null(h_last))
    return MMF_ERR_ALIGN;
  return MMF_OK;
}

size_t scan_ws_bytes(int64_t B, int64_t T, int64_t d) {
  return round_up(static_cast<size_t>(mmf::mlgru_scan_ws_floats(B, T, d)) * 4, kScratchAlign);
}

// Scratch of the whole mixer: fcg [M][3d], o' [M][d], the quantised
// activations of either projection, the scan's chunk summaries.
struct MlgruScratch {
  size_t fcg_off, op_off, q_off, scan_off, total;
};
MlgruScratch mlgru_scratch(int64_t B, int64_t T, int64_t d) {
  const size_t M = static_cast<size_t>(B) * static_cast<size_t>(T);
  MlgruScratch s;
  s.fcg_off = 0;
  s.op_off = round_up(M * 3 * static_cast<size_t>(d) * 4, kScratchAlign);
  s.q_off = s.op_off + round_up(M * static_cast<size_t>(d) * 4, kScratchAlign);
  s.scan_off = s.q_off + fwd_scratch(static_cast<int64_t>(M), d).total;
  s.total = s.scan_off + scan_ws_bytes(B, T, d);
  return s;
}

// ---- training forward and backward ----

struct TrainScratch {
  size_t part_off, rs_off, total;
};
TrainScratch train_scratch(int64_t M, int64_t K, int64_t N) {
  TrainScratch s;
  s.part_off = 0;
  s.rs_off = round_up(sizeof(double) * static_cast<size_t>(mmf::ternarize_partials_count(N * K)), kScratchAlign);
  s.total = s.rs_off + round_up(static_cast<size_t>(M) * 4, kScratchAlign);
  return s;
}


struct BwdScratch {
  int64_t Np;
  mmf::DwPlan plan;
  size_t wn_off, dop_off, spart_off, dgpart_off, dbpart_off, dw_off, parts_off, total;
};
BwdScratch bwd_scratch(int64_t M, int64_t K, int64_t N) {
  BwdScratch s;
  s.Np = (N + 7) / 8 * 8;
  s.plan = mmf::bwd_dw_plan(M, N, K, s.Np, mmf::device_cus());
  s.wn_off = 0;
  s.dop_off = round_up(static_cast<size_t>(mmf::bwd_nmajor_words(N, K)) * 4, kScratchAlign);
  const size_t dop = s.Np != N ? static_cast<size_t>(M) * static_cast<size_t>(s.Np) * 2 : 0;
  s.spart_off = s.dop_off + round_up(dop, kScratchAlign);
  s.dgpart_off = s.spart_off + round_up(sizeof(double) * static_cast<size_t>(mmf::bwd_dy_col_tiles(K) * M),
                                        kScratchAlign);
  s.dbpart_off = s.dgpart_off + round_up(sizeof(double) * static_cast<size_t>(mmf::bwd_dy_row_tiles(M) * K),
                                          kScratchAlign);
  s.dw_off = s.dbpart_off + round_up(sizeof(double) * static_cast<size_t>(mmf::bwd_dy_row_tiles(M) * N),
                                      kScratchAlign);
  const int64_t S = s.plan.split_all;
  s.parts_off = s.dw_off + (S > 1 ? round_up(sizeof(float) * static_cast<size_t>(S * N * K), kScratchAlign) : 0);
  s.total = s.parts_off + round_up(mmf::bwd_dw_parts_bytes(s.plan), kScratchAlign);
  return s;
}

// Shapes the backward's kernels address with 32-bit offsets: the n-major
// codes and the dY launch's dO rows (bwd_dy_row_slice), dW [N][K] and the
// token counts.
int check_bwd_shape(int64_t M, int64_t K, int64_t N) {
  const int64_t lim = (int64_t(1) << 31) - 1;
  const int64_t Np = (N + 7) / 8 * 8;
  if (mmf::bwd_dy_row_slice(Np, K) == 0 || N * K * 4 > lim || M > lim) return MMF_ERR_SHAPE;
  return MMF_OK;
}

// ---- the forward without allocation (mmf_bitlinear_fwd_noalloc) ----
//
// Its scratch (q, a_scale, q_rowsum: fwd_scratch) lives in a file-scope
// device array, one copy per GPU, held until the process ends.  Host code
// never passes the array's name to a kernel (on the host that name is only a
// stand-in, not a device address): the address of each device's copy comes
// from hipGetSymbolAddress, taken once per device with that device current
// (on the entry point's first call there), and is used everywhere after.
constexpr size_t kNoAllocScratchBytes = size_t(64) << 20;
__device__ __align__(256) char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch`, or nullptr (with *status set) when
// the device cannot be determined or the address lookup fails.
char* device_scratch(int* status) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    *status = MMF_ERR_HIP;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) {
      *status = MMF_ERR_HIP;
      return nullptr;
    }
    g_scratch_ptr[dev] = static_cast<char*>(p);
  }
  return g_scratch_ptr[dev];
}

}  // namespace

// Compute units of the current device, cached per device (the work plans of
// the dW kernel and the tile choice of the MFMA contraction).
int mmf::device_cus() {
  static std::mutex mu;
  static int cus[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  std::lock_guard<std::mutex> lock(mu);
  if (cus[dev] == 0) {
    int v = 0;
    cus[dev] = (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0) ? v : 256;
  }
  return cus[dev];
}

extern "C" {

const char* mmf_status_string(int status) {
  switch (status) {
    case MMF_OK: return "MMF_OK";
    case MMF_ERR_NULL: return "MMF_ERR_NULL: a required pointer is NULL";
    case MMF_ERR_SHAPE: return "MMF_ERR_SHAPE: size out of range (K must be a positive multiple of 16, at most 2^20; M, N in [0, 2^31-1]; the kernel's 32-bit offset limits)";
    case MMF_ERR_ALIGN: return "MMF_ERR_ALIGN: an array pointer is not 16-byte aligned";
    case MMF_ERR_DTYPE: return "MMF_ERR_DTYPE: the activation dtype selector must be 0 (bf16) or 1 (float32)";
    case MMF_ERR_HIP: return "MMF_ERR_HIP: a HIP runtime call or kernel launch failed";
    case MMF_ERR_WORKSPACE: return "MMF_ERR_WORKSPACE: workspace too small or misaligned";
    case MMF_ERR_ARG: return "MMF_ERR_ARG: invalid argument";
    default: return "MMF: unknown status";
  }
}

int mmf_version(void) { return 2; }

size_t mmf_packed_weight_bytes(int64_t N, int64_t K) {
  if (check_shape(0, K, N) != MMF_OK) return 0;
  return static_cast<size_t>(K / 16) * static_cast<size_t>(N) * 4u;
}

int mmf_ternarize_weights(const float* W, int64_t N, int64_t K, uint32_t* Wpacked,
                          float* w_scale, hipStream_t stream) {
  if (int st = check_shape(0, K, N)) return st;
  if (N == 0) return MMF_OK;
  if (!W || !Wpacked || !w_scale) return MMF_ERR_NULL;
  if (!aligned16(W) || !aligned16(Wpacked)) return MMF_ERR_ALIGN;
  const int n_part = mmf::ternarize_partials_count(N * K);
  void* partials = nullptr;
  if (hipMallocAsync(&partials, sizeof(double) * n_part, stream) != hipSuccess) return MMF_ERR_HIP;
  const hipError_t e = mmf::launch_ternarize(W, N, static_cast<int>(K), Wpacked, w_scale,
                                             static_cast<double*>(partials), stream);
  const hipError_t fe = hipFreeAsync(partials, stream);
  if (e != hipSuccess) return MMF_ERR_HIP;
  return hip_status(fe);
}

int mmf_act_quant(const uint16_t* x, const float* gamma, int8_t* q, float* a_scale, int64_t M,
                  int64_t K, hipStream_t stream) {
  return act_quant_common(x, 0, gamma, q, a_scale, nullptr, M, K, stream);
}

int mmf_act_quant_f32(const float* x, const float* gamma, int8_t* q, float* a_scale, int64_t M,
                      int64_t K, hipStream_t stream) {
  return act_quant_common(x, 1, gamma, q, a_scale, nullptr, M, K, stream);
}

int mmf_act_quant_ex(const void* x, int x_is_f32, const float* gamma, int8_t* q, float* a_scale,
                     int32_t* q_rowsum, int64_t M, int64_t K, hipStream_t stream) {
  return act_quant_common(x, x_is_f32, gamma, q, a_scale, q_rowsum, M, K, stream);
}

int mmf_bitlinear_fwd(const uint16_t* x, const float* gamma, const uint32_t* Wpacked,
                      const float* w_scale, float* y, int64_t M, int64_t K, int64_t N,
                      hipStream_t stream) {
  return fwd_alloc(x, false, gamma, Wpacked, w_scale, y, M, K, N, stream);
}

int mmf_bitlinear_fwd_f32(const float* x, const float* gamma, const uint32_t* Wpacked,
                          const float* w_scale, float* y, int64_t M, int64_t K, int64_t N,
                          hipStream_t stream) {
  return fwd_alloc(x, true, gamma, Wpacked, w_scale, y, M, K, N, stream);
}

size_t mmf_bitlinear_workspace_bytes(int64_t M, int64_t K) {
  if (check_shape(M, K, 0) != MMF_OK) return 0;
  return fwd_scratch(M, K).total;
}

int mmf_bitlinear_fwd_ws(const void* x, int x_is_f32, const float* gamma,
                         const uint32_t* Wpacked, const float* w_scale, float* y, int64_t M,
                         int64_t K, int64_t N, void* workspace, size_t workspace_bytes,
                         hipStream_t stream) {
  if (int st = check_dtype(x_is_f32)) return st;
  if (int st = check_fwd(x, x_is_f32 == 1, gamma, Wpacked, w_scale, y, M, K, N)) return st;
  if (M == 0 || N == 0) return MMF_OK;
  if (!workspace) return MMF_ERR_NULL;
  if ((reinterpret_cast<uintptr_t>(workspace) & (kScratchAlign - 1)) != 0 ||
      workspace_bytes < fwd_scratch(M, K).total)
    return MMF_ERR_WORKSPACE;
  return run_fwd(x, x_is_f32 == 1, gamma, Wpacked, w_scale, y, M, K, N,
                 static_cast<char*>(workspace), stream);
}

size_t mmf_bitlinear_noalloc_max_bytes(void) { return kNoAllocScratchBytes; }

int mmf_bitlinear_fwd_noalloc(const void* x, int x_is_f32, const float* gamma,
                              const uint32_t* Wpacked, const float* w_scale, float* y, int64_t M,
                              int64_t K, int64_t N, hipStream_t stream) {
  if (int st = check_dtype(x_is_f32)) return st;
  if (int st = check_fwd(x, x_is_f32 == 1, gamma, Wpacked, w_scale, y, M, K, N)) return st;
  if (M == 0 || N == 0) return MMF_OK;
  const bool f32 = x_is_f32 == 1;
  // few tokens: fused decode launches, which use no scratch
  if (fused_decode(M, K, N, f32))
    return hip_status(run_fused_decode(x, f32, gamma, Wpacked, w_scale, y, M, K, N, stream));
  if (fwd_scratch(M, K).total > kNoAllocScratchBytes) return MMF_ERR_WORKSPACE;
  int st = MMF_OK;
  char* ws = device_scratch(&st);
  if (ws == nullptr) return st;
  return run_fwd(x, f32, gamma, Wpacked, w_scale, y, M, K, N, ws, stream);
}

int mmf_ternary_gemm_dequant(const int8_t* q, const float* a_scale, const int32_t* q_rowsum,
                             const uint32_t* Wpacked, const float* w_scale, float* y, int64_t M,
                             int64_t K, int64_t N, hipStream_t stream) {
  if (int st = check_shape(M, K, N)) return st;
  if (M == 0 || N == 0) return MMF_OK;
  if (int st = check_contract(M, K, N)) return st;
  if (!q || !a_scale || !q_rowsum || !Wpacked || !w_scale || !y) return MMF_ERR_NULL;
  if (!aligned16(q) || !aligned16(a_scale) || !aligned16(q_rowsum) || !aligned16(Wpacked) ||
      !aligned16(y))
    return MMF_ERR_ALIGN;
  mmf::ContractArgs a{q, a_scale, q_rowsum, Wpacked, w_scale, y, M, static_cast<int>(K), N,
                      mmf::Epilogue::kDequantF32};
  return hip_status(contract(a, stream));
}

int mmf_ternary_gemm_i32(const int8_t* q, const uint32_t* Wpacked, int32_t* acc, int64_t M,
                         int64_t K, int64_t N, hipStream_t stream) {
  if (int st = check_shape(M, K, N)) return st;
  if (M == 0 || N == 0) return MMF_OK;
  if (int st = check_contract(M, K, N)) return st;
  if (!q || !Wpacked || !acc) return MMF_ERR_NULL;
  if (!aligned16(q) || !aligned16(Wpacked) || !aligned16(acc)) return MMF_ERR_ALIGN;
  void* rowsum = nullptr;
  if (hipMallocAsync(&rowsum, round_up(static_cast<size_t>(M) * 4, kScratchAlign), stream) !=
      hipSuccess)
    return MMF_ERR_HIP;
  int32_t* rs = static_cast<int32_t*>(rowsum);
  hipError_t e = mmf::launch_row_sum(q, rs, M, static_cast<int>(K), stream);
  if (e == hipSuccess) {
    mmf::ContractArgs a{q, nullptr, rs, Wpacked, nullptr, acc, M, static_cast<int>(K), N,
                        mmf::Epilogue::kRawI32};
    e = contract(a, stream);
  }
  const hipError_t fe = hipFreeAsync(rowsum, stream);
  if (e != hipSuccess) return MMF_ERR_HIP;
  return hip_status(fe);
}

int mmf_glu_pack(const uint32_t* Wg_packed, const uint32_t* Wu_packed, int64_t L, int64_t K,
                 uint32_t* Wgu_packed, hipStream_t stream) {
  if (L < 0 || L > kMaxMN / 2 || (L % 16) != 0) return MMF_ERR_SHAPE;
  if (int st = check_shape(0, K, 2 * L)) return st;
  if (L == 0) return MMF_OK;
  if (!Wg_packed || !Wu_packed || !Wgu_packed) return MMF_ERR_NULL;
  if (!aligned16(Wg_packed) || !aligned16(Wu_packed) || !aligned16(Wgu_packed)) return MMF_ERR_ALIGN;
  return hip_status(mmf::launch_glu_pack(Wg_packed, Wu_packed, L, static_cast<int>(K), Wgu_packed, stream));
}

int mmf_glu_fwd(const uint16_t* x, const float* gamma, const uint32_t* Wgu_packed,
                const float* w_scales, float* p, int64_t M, int64_t K, int64_t L,
                hipStream_t stream) {
  return glu_alloc(x, false, gamma, Wgu_packed, w_scales, p, M, K, L, stream);
}

int mmf_glu_fwd_f32(const float* x, const float* gamma, const uint32_t* Wgu_packed,
                    const float* w_scales, float* p, int64_t M, int64_t K, int64_t L,
                    hipStream_t stream) {
  return glu_alloc(x, true, gamma, Wgu_packed, w_scales, p, M, K, L, stream);
}

int mmf_glu_fwd_ws(const void* x, int x_is_f32, const float* gamma, const uint32_t* Wgu_packed,
                   const float* w_scales, float* p, int64_t M, int64_t K, int64_t L,
                   void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (int st = check_dtype(x_is_f32)) return st;
  if (int st = check_glu(x, x_is_f32 == 1, gamma, Wgu_packed, w_scales, p, M, K, L)) return st;
  if (M == 0 || L == 0) return MMF_OK;
  if (!workspace) return MMF_ERR_NULL;
  if ((reinterpret_cast<uintptr_t>(workspace) & (kScratchAlign - 1)) != 0 ||
      workspace_bytes < fwd_scratch(M, K).total)
    return MMF_ERR_WORKSPACE;
  return run_glu(x, x_is_f32 == 1, gamma, Wgu_packed, w_scales, p, M, K, L,
                 static_cast<char*>(workspace), stream);
}

int mmf_ternary_gemm_glu(const int8_t* q, const float* a_scale, const int32_t* q_rowsum,
                         const uint32_t* Wgu_packed, const float* w_scales, float* p, int64_t M,
                         int64_t K, int64_t L, hipStream_t stream) {
  if (L < 0 || L > kMaxMN / 2 || (L % 16) != 0) return MMF_ERR_SHAPE;
  if (int st = check_shape(M, K, 2 * L)) return st;
  if (M == 0 || L == 0) return MMF_OK;
  if (int st = check_gemm(K, 2 * L)) return st;
  if (!q || !a_scale || !q_rowsum || !Wgu_packed || !w_scales || !p) return MMF_ERR_NULL;
  if (!aligned16(q) || !aligned16(a_scale) || !aligned16(q_rowsum) || !aligned16(Wgu_packed) ||
      !aligned16(p))
    return MMF_ERR_ALIGN;
  mmf::ContractArgs a{q, a_scale, q_rowsum, Wgu_packed, w_scales, p, M, static_cast<int>(K), 2 * L,
                      mmf::Epilogue::kGluF32};
  return hip_status(mmf::launch_gemm(a, stream));
}

int mmf_bitlinear_fwd_bias(const void* x, int x_is_f32, const float* gamma,
                           const uint32_t* Wpacked, const float* w_scale, const float* bias,
                           float* y, int64_t M, int64_t K, int64_t N, hipStream_t stream) {
  if (int st = check_dtype(x_is_f32)) return st;
  if (int st = check_fwd(x, x_is_f32 == 1, gamma, Wpacked, w_scale, y, M, K, N, true)) return st;
  if (N % 4 != 0) return MMF_ERR_SHAPE;
  if (M == 0 || N == 0) return MMF_OK;
  if (!bias) return MMF_ERR_NULL;
  if (!aligned16(bias)) return MMF_ERR_ALIGN;
  mmf::Affine aff;
  aff.bias = bias;
  aff.seg = N;
  aff.acts = mmf::kActIdentity;
  const size_t need = fused_decode(M, K, N, x_is_f32 == 1) ? 0 : fwd_scratch(M, K).total;
  return with_workspace(nullptr, 0, need, stream, [&](char* scratch) {
    return run_affine(x, x_is_f32 == 1, gamma, Wpacked, w_scale, aff, y, M, K, N, scratch, stream);
  });
}

size_t mmf_mlgru_proj_workspace_bytes(int64_t M, int64_t K, int64_t d) {
  if (check_mlgru_d(d) != MMF_OK || check_shape(M, K, 3 * d) != MMF_OK) return 0;
  return fwd_scratch(M, K).total;
}

int mmf_mlgru_proj(const void* x, int x_is_f32, const float* gamma, const uint32_t* Wfcg,
                   const float* w_scales, const float* bias, const float* lb, float* fcg,
                   int64_t M, int64_t K, int64_t d, void* workspace, size_t workspace_bytes,
                   hipStream_t stream) {
  if (int st = check_dtype(x_is_f32)) return st;
  if (int st = check_mlgru_proj(x, gamma, Wfcg, w_scales, bias, lb, fcg, M, K, d)) return st;
  if (M == 0) return MMF_OK;
  if (int st = check_from_x(M, K, 3 * d, x_is_f32 == 1, true)) return st;
  mmf::Affine aff;
  aff.bias = bias;
  aff.lb = lb;
  aff.seg = d;
  aff.acts = kMlgruActs;
  return with_workspace(workspace, workspace_bytes, fwd_scratch(M, K).total, stream, [&](char* scratch) {
    return run_affine(x, x_is_f32 == 1, gamma, Wfcg, w_scales, aff, fcg, M, K, 3 * d, scratch, stream);
  });
}

int mmf_mlgru_proj_q(const int8_t* q, const float* a_scale, const int32_t* q_rowsum,
                     const uint32_t* Wfcg, const float* w_scales, const float* bias,
                     const float* lb, float* fcg, int64_t M, int64_t K, int64_t d,
                     hipStream_t stream) {
  if (int st = check_mlgru_d(d)) return st;
  if (int st = check_shape(M, K, 3 * d)) return st;
  if (M == 0) return MMF_OK;
  if (int st = check_gemm(K, 3 * d)) return st;
  if (!q || !a_scale || !q_rowsum || !Wfcg || !w_scales || !fcg) return MMF_ERR_NULL;
  if (!aligned16(q) || !aligned16(a_scale) || !aligned16(q_rowsum) || !aligned16(Wfcg) ||
      !aligned16(fcg) || !aligned16_or_null(bias) || !aligned16_or_null(lb))
    return MMF_ERR_ALIGN;
  mmf::Affine aff;
  aff.bias = bias;
  aff.lb = lb;
  aff.seg = d;
  aff.acts = kMlgruActs;
  mmf::ContractArgs a{q, a_scale, q_rowsum, Wfcg, w_scales, fcg, M, static_cast<int>(K), 3 * d,
                      mmf::Epilogue::kAffineF32, aff};
  return hip_status(mmf::launch_gemm(a, stream));
}

size_t mmf_mlgru_scan_workspace_bytes(int64_t B, int64_t T, int64_t d) {
  if (check_mlgru_d(d) != MMF_OK || B < 0 || T < 0) return 0;
  return scan_ws_bytes(B, T, d);
}

int mmf_mlgru_scan(const float* fcg, const float* h0, float* o_prime, float* h_last, int64_t B,
                   int64_t T, int64_t d, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (int st = check_mlgru_scan(fcg, h0, o_prime, h_last, B, T, d)) return st;
  if (B == 0 || T == 0) return MMF_OK;
  return with_workspace(workspace, workspace_bytes, scan_ws_bytes(B, T, d), stream, [&](char* scratch) {
    return hip_status(mmf::launch_mlgru_scan(fcg, h0, o_prime, h_last, B, T, d,
                                             reinterpret_cast<float*>(scratch), stream));
  });
}

size_t mmf_mlgru_workspace_bytes(int64_t B, int64_t T, int64_t d) {
  if (check_mlgru_d(d) != MMF_OK || B < 0 || T < 0 || (T > 0 && B > kMaxMN / T)) return 0;
  return mlgru_scratch(B, T, d).total;
}

int mmf_mlgru_fwd(const void* x, int x_is_f32, const float* gamma, const uint32_t* Wfcg,
                  const float* w_scales, const float* bias, const float* lb, const float* h0,
                  float* h_last, const float* gamma_o, const uint32_t* Wo, const float* w_scale_o,
                  const float* b_o, float* o, int64_t B, int64_t T, int64_t d, void* workspace,
                  size_t workspace_bytes, hipStream_t stream) {
  if (int st = check_dtype(x_is_f32)) return st;
  if (int st = check_mlgru_d(d)) return st;
  if (d > kMaxK) return MMF_ERR_SHAPE;
  if (B < 0 || T < 0 || B > kMaxMN || T > kMaxMN || (T > 0 && B > kMaxMN / T)) return MMF_ERR_SHAPE;
  const int64_t M = B * T;
  if (M == 0) return MMF_OK;
  if (int st = check_from_x(M, d, 3 * d, x_is_f32 == 1, true)) return st;
  if (int st = check_from_x(M, d, d, true, true)) return st;
  if (!x || !Wfcg || !w_scales || !Wo || !w_scale_o || !o) return MMF_ERR_NULL;
  if (!aligned16(x) || !aligned16(Wfcg) || !aligned16(Wo) || !aligned16(o) ||
      !aligned16_or_null(gamma) || !aligned16_or_null(bias) || !aligned16_or_null(lb) ||
      !aligned16_or_null(h0) || !aligned16_or_null(h_last) || !aligned16_or_null(gamma_o) ||
      !aligned16_or_null(b_o))
    return MMF_ERR_ALIGN;
  const MlgruScratch s = mlgru_scratch(B, T, d);
  return with_workspace(workspace, workspace_bytes, s.total, stream, [&](char* scratch) {
    float* fcg = reinterpret_cast<float*>(scratch + s.fcg_off);
    float* op = reinterpret_cast<float*>(scratch + s.op_off);
    mmf::Affine in;
    in.bias = bias;
    in.lb = lb;
    in.seg = d;
    in.acts = kMlgruActs;
    int st = run_affine(x, x_is_f32 == 1, gamma, Wfcg, w_scales, in, fcg, M, d, 3 * d,
                        scratch + s.q_off, stream);
    if (st != MMF_OK) return st;
    mmf::Affine out;
    out.bias = b_o;
    out.seg = d;
    out.acts = mmf::kActIdentity;
    // A decode step (one token per sequence) with the new state in its own
    // array: the recurrence and output gate run in the output projection's
    // prologue (no launch, no o' round trip).  Identical arithmetic to the
    // separate kernels, so identical results.
    if (T == 1 && (h_last == nullptr || h_last != h0) && fused_decode(M, d, d, true)) {
      for (int64_t m0 = 0; m0 < M; m0 += kDecodeMaxTokens) {
        const int64_t mt = M - m0 < kDecodeMaxTokens ? M - m0 : kDecodeMaxTokens;
        mmf::DecodeArgs a{fcg + m0 * 3 * d, true, gamma_o, nullptr, nullptr, nullptr, Wo, w_scale_o,
                          o + m0 * d, mt, static_cast<int>(d), d, mmf::Epilogue::kAffineF32, out};
        a.mlgru_in = true;
        a.h_in = h0 ? h0 + m0 * d : nullptr;
        a.h_out = h_last ? h_last + m0 * d : nullptr;
        if (mmf::launch_decode(a, stream) != hipSuccess) return MMF_ERR_HIP;
      }
      return MMF_OK;
    }
    if (mmf::launch_mlgru_scan(fcg, h0, op, h_last, B, T, d, reinterpret_cast<float*>(scratch + s.scan_off),
                               stream) != hipSuccess)
      return MMF_ERR_HIP;
    return run_affine(op, true, gamma_o, Wo, w_scale_o, out, o, M, d, d, scratch + s.q_off, stream);
  });
}

size_t mmf_bitlinear_train_workspace_bytes(int64_t M, int64_t K, int64_t N) {
  if (check_shape(M, K, N) != MMF_OK) return 0;
  return train_scratch(M, K, N).total;
}

int mmf_bitlinear_train_fwd(const void* x, int x_is_f32, const float* gamma, const float* W,
                            const float* bias, float* y, uint32_t* Wpacked, float* w_scale, int8_t* q,
                            float* a_scale, float* rstd, int64_t M, int64_t K, int64_t N, void* workspace,
                            size_t workspace_bytes, hipStream_t stream) {
  if (int st = check_dtype(x_is_f32)) return st;
  if (int st = check_shape(M, K, N)) return st;
  if (check_gemm(K, N) != MMF_OK || (bias && N % 4 != 0)) return MMF_ERR_SHAPE;
  if (M == 0 || N == 0) return MMF_OK;
  if (!x || !W || !y || !Wpacked || !w_scale || !q || !a_scale) return MMF_ERR_NULL;
  if (!aligned16(x) || !aligned16(W) || !aligned16(y) || !aligned16(Wpacked) || !aligned16(q) ||
      !aligned16(a_scale) || !aligned16_or_null(gamma) || !aligned16_or_null(bias) || !aligned16_or_null(rstd))
    return MMF_ERR_ALIGN;
  const TrainScratch s = train_scratch(M, K, N);
  return with_workspace(workspace, workspace_bytes, s.total, stream, [&](char* scratch) {
    int32_t* rowsum = reinterpret_cast<int32_t*>(scratch + s.rs_off);
    if (mmf::launch_ternarize(W, N, static_cast<int>(K), Wpacked, w_scale,
                              reinterpret_cast<double*>(scratch + s.part_off), stream) != hipSuccess)
      return MMF_ERR_HIP;
    if (mmf::launch_act_quant(x, x_is_f32 == 1, gamma, q, a_scale, rowsum, M, static_cast<int>(K), stream,
                              rstd) != hipSuccess)
      return MMF_ERR_HIP;
    mmf::Affine aff;
    aff.bias = bias;
    aff.seg = N;
    aff.acts = mmf::kActIdentity;
    mmf::ContractArgs a{q, a_scale, rowsum, Wpacked, w_scale, y, M, static_cast<int>(K), N,
                        bias ? mmf::Epilogue::kAffineF32 : mmf::Epilogue::kDequantF32, aff};
    return hip_status(mmf::launch_gemm(a, stream));
  });
}

size_t mmf_bitlinear_bwd_workspace_bytes(int64_t M, int64_t K, int64_t N) {
  if (check_shape(M, K, N) != MMF_OK || check_bwd_shape(M, K, N) != MMF_OK) return 0;
  return bwd_scratch(M, K, N).total;
}

int mmf_bitlinear_bwd(const uint16_t* dO, const void* x, int x_is_f32, const float* gamma,
                      const float* rstd, const int8_t* q, const float* a_scale, const uint32_t* Wpacked,
                      const float* w_scale, float* dx, float* dW, float* db, float* dgamma, int64_t M,
                      int64_t K, int64_t N, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (int st = check_dtype(x_is_f32)) return st;
  if (int st = check_shape(M, K, N)) return st;
  if (int st = check_bwd_shape(M, K, N)) return st;
  if (M == 0 || N == 0) return MMF_OK;
  if (!dO || !x || !rstd || !q || !a_scale || !Wpacked || !w_scale || !dx || !dW) return MMF_ERR_NULL;
  if (!aligned16(dO) || !aligned16(x) || !aligned16(rstd) || !aligned16(q) || !aligned16(a_scale) ||
      !aligned16(Wpacked) || !aligned16(dx) || !aligned16(dW) || !aligned16_or_null(gamma) ||
      !aligned16_or_null(db) || !aligned16_or_null(dgamma))
    return MMF_ERR_ALIGN;
  const BwdScratch s = bwd_scratch(M, K, N);
  return with_workspace(workspace, workspace_bytes, s.total, stream, [&](char* scratch) {
    uint32_t* Wn = reinterpret_cast<uint32_t*>(scratch + s.wn_off);
    double* s_part = reinterpret_cast<double*>(scratch + s.spart_off);
    double* dg_part = dgamma ? reinterpret_cast<double*>(scratch + s.dgpart_off) : nullptr;
    const int Ki = static_cast<int>(K);
    const bool f32 = x_is_f32 == 1;
    // dO rows in 16-byte chunks: zero-padded copy when N % 8 != 0
    const uint16_t* dOp = dO;
    if (s.Np != N) {
      uint16_t* pad = reinterpret_cast<uint16_t*>(scratch + s.dop_off);
      if (mmf::launch_pad_rows(dO, M, N, s.Np, pad, stream) != hipSuccess) return MMF_ERR_HIP;
      dOp = pad;
    }
    // dY = dO Wt^T with r gamma dY into dx and the row / column partials,
    // then dx and dgamma finished
    if (mmf::launch_pack_nmajor(Wpacked, N, s.Np, Ki, Wn, stream) != hipSuccess) return MMF_ERR_HIP;
    double* db_part = db ? reinterpret_cast<double*>(scratch + s.dbpart_off) : nullptr;
    if (mmf::launch_dy(dOp, M, N, s.Np, Wn, w_scale, x, f32, gamma, rstd, Ki, dx, s_part, dg_part, db_part,
                       stream) != hipSuccess)
      return MMF_ERR_HIP;
    if (mmf::launch_dx_finish(dx, x, f32, rstd, s_part, M, Ki, stream) != hipSuccess) return MMF_ERR_HIP;
    if (dgamma && mmf::launch_dgamma_finish(dg_part, M, Ki, dgamma, stream) != hipSuccess) return MMF_ERR_HIP;
    // dW = dO^T Yq (token range split into parts when the output has few
    // tiles; the last partial round of tiles spread over all CUs otherwise)
    const int64_t S = s.plan.split_all;
    float* dw_out = S > 1 ? reinterpret_cast<float*>(scratch + s.dw_off) : dW;
    float* parts = s.plan.tail_units > 0 ? reinterpret_cast<float*>(scratch + s.parts_off) : nullptr;
    if (mmf::launch_dw(dOp, q, a_scale, M, s.Np, N, Ki, dw_out, parts, s.plan, stream) != hipSuccess)
      return MMF_ERR_HIP;
    if (S > 1 && mmf::launch_sum_parts(dw_out, S, N * K, dW, stream) != hipSuccess) return MMF_ERR_HIP;
    if (db && mmf::launch_db_finish(db_part, M, N, db, stream) != hipSuccess) return MMF_ERR_HIP;
    return MMF_OK;
  });
}

int mmf_set_path(int path) {
  if (path != MMF_PATH_AUTO && path != MMF_PATH_GEMV && path != MMF_PATH_GEMM)
    return -MMF_ERR_ARG;
  return g_path.exchange(path);
}

static_assert(mmf::kPlan128x512 == MMF_TILE_128x512 && mmf::kPlan128x256Paired == MMF_TILE_128x256_PAIRED &&
                  mmf::kPlan64x512 == MMF_TILE_64x512 && mmf::kPlan64x256 == MMF_TILE_64x256 &&
                  mmf::kPlan256x256 == MMF_TILE_256x256,
              "tile plan values follow the header");

int mmf_prefill_tile_plan(int64_t M, int64_t K, int64_t N, int epilogue, int cus) {
  if (const int st = check_shape(M, K, N); st != MMF_OK) return -st;
  if (M < 1 || N < 1 || cus < 1 || check_gemm(K, N) != MMF_OK) return -MMF_ERR_SHAPE;
  mmf::Epilogue ep;
  switch (epilogue) {
    case MMF_EPILOGUE_DEQUANT: ep = mmf::Epilogue::kDequantF32; break;
    case MMF_EPILOGUE_RAW_I32: ep = mmf::Epilogue::kRawI32; break;
    case MMF_EPILOGUE_GLU: ep = mmf::Epilogue::kGluF32; break;
    case MMF_EPILOGUE_AFFINE: ep = mmf::Epilogue::kAffineF32; break;
    default: return -MMF_ERR_ARG;
  }
  if (ep == mmf::Epilogue::kGluF32 && N % 32 != 0) return -MMF_ERR_SHAPE;
  const int64_t slice = mmf::gemm_row_slice(K, N);
  return mmf::gemm_plan(M < slice ? M : slice, static_cast<int>(K), N, ep, cus);
}

}  // extern "C"
