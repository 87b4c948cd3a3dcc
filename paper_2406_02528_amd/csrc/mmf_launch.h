// Internal launchers of the gfx950 kernels.  Shapes are validated by the
// C-ABI layer before any of these is called.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mmf {

// RMSNorm + absmax int8 quantisation of M rows of K features (K % 16 == 0);
// rstd (optional) receives each row's 1/sqrt(mean x^2 + eps).
hipError_t launch_act_quant(const void* x, bool x_is_f32, const float* gamma, int8_t* q,
                            float* a_scale, int32_t* q_rowsum, int64_t M, int K,
                            hipStream_t stream, float* rstd = nullptr);

// q_rowsum[m] = sum_k q[m][k].
hipError_t launch_row_sum(const int8_t* q, int32_t* q_rowsum, int64_t M, int K,
                          hipStream_t stream);

// Ternarisation: partial sums of |W| (fp64), finalise w_scale, pack.
// `partials` must hold ternarize_partials_count(N*K) doubles.
int ternarize_partials_count(int64_t count);
hipError_t launch_ternarize(const float* W, int64_t N, int K, uint32_t* Wpacked,
                            float* w_scale, double* partials, hipStream_t stream);

// Output form of the contraction kernels.  kGluF32: the packed columns are
// the two up-projections of a GLU interleaved in blocks of 16 (gate, up,
// gate, ...), w_scale holds [gate, up], and the output is the gated
// representation SiLU(g) * u, N / 2 columns wide.
enum class Epilogue { kDequantF32, kRawI32, kGluF32, kAffineF32 };

// kAffineF32: y = act_s(acc * a_scale * w_scale[s] + bias[n]) with the columns
// in segments of `seg` (s = n / seg, seg % 16 == 0) and one activation per
// segment, 2 bits each in `acts` (segment s at bits 2s, 2s + 1):
//   kActIdentity  y = z
//   kActSigmoidLb y = lb + (1 - lb) sigmoid(z), lb = lb[n % seg] (0 if null)
//   kActSilu      y = z sigmoid(z)
// bias may be null (no bias).  At most 16 segments.
constexpr uint32_t kActIdentity = 0, kActSigmoidLb = 1, kActSilu = 2;
struct Affine {
  const float* bias = nullptr;  // [N]
  const float* lb = nullptr;    // [seg]
  int64_t seg = 0;
  uint32_t acts = 0;
};

struct ContractArgs {
  const int8_t* q;          // [M][K]
  const float* a_scale;     // [M]   (kDequantF32 only)
  const int32_t* q_rowsum;  // [M]
  const uint32_t* Wpacked;  // [K/16][N]
  const float* w_scale;     // [1]   (kDequantF32 only)
  void* out;                // [M][N] float or int32
  int64_t M;
  int K;
  int64_t N;
  Epilogue epilogue;
  Affine affine{};          // kAffineF32 only; w_scale then holds N / seg values
};

// Decode contraction with q read from global memory (scalar loads); any K,
// M <= 8 per launch (larger M is sliced).
hipError_t launch_gemv(const ContractArgs& a, hipStream_t stream);

// Fused decode forward: up to 16 tokens per launch, q kept in LDS (the q
// region of M rows of K + 16 bytes, in whole KB, at most kDecodeMaxLdsQ).
// With q == nullptr it normalises and quantises x itself; otherwise it
// contracts the given q / a_scale / q_rowsum.
constexpr int kDecodeMaxTokens = 16;
constexpr int kDecodeMaxLdsQ = 131072;
struct DecodeArgs {
  const void* x;            // [M][K] bf16 or f32 (q == nullptr)
  bool x_is_f32;
  const float* gamma;       // [K] or nullptr
  const int8_t* q;          // [M][K] or nullptr
  const float* a_scale;     // [M] (q path, dequant epilogue)
  const int32_t* q_rowsum;  // [M] (q path)
  const uint32_t* Wpacked;  // [K/16][N]
  const float* w_scale;     // [1]
  void* out;                // [M][N]
  int64_t M;                // 1..kDecodeMaxTokens
  int K;
  int64_t N;
  Epilogue epilogue;
  Affine affine{};          // kAffineF32 only
  // MLGRU output projection (kAffineF32): x is the gates fcg [M][3K] and the
  // activations are o' = g sigmoid(f h + (1 - f) c) with h = h_in [M][K]
  // (nullptr: 0); the new state goes to h_out (nullptr: not stored), which
  // must not be h_in (every workgroup reads all of h_in).
  bool mlgru_in = false;
  const float* h_in = nullptr;
  float* h_out = nullptr;
};
bool decode_fits(int64_t mt, int K, int64_t N, bool from_x, bool x_is_f32);
hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream);
// Compute units of the current device (cached per device).
int device_cus();
// Prefill kernel: int8 MFMA, any M.  The workgroup tile is 128 x 512, or
// 64 x 512 / 64 x 256 when those finish a problem with few 128 x 512 tiles
// sooner (gemm_tile_choice); 256 x 256 when N % 4 != 0.  Where 128 x 512 is
// chosen at K <= 4096 it runs as two 128 x 256 workgroups per CU once its
// tiles fill the CUs (except with the affine epilogue).
hipError_t launch_gemm(const ContractArgs& a, hipStream_t stream);
// Index of the tile shape launch_gemm uses for `rows` x N on `cus` compute
// units (N % 4 == 0): 0 for 128 x 512, 1 for 64 x 512, 2 for 64 x 256.
int gemm_tile_choice(int64_t rows, int64_t N, int cus);
// The tile plan launch_gemm follows for one launch of `rows` x K x N with
// epilogue `ep` on `cus` compute units (the values of MMF_TILE_* in mmf.h).
enum GemmPlan { kPlan128x512 = 0, kPlan128x256Paired = 1, kPlan64x512 = 2, kPlan64x256 = 3, kPlan256x256 = 4 };
int gemm_plan(int64_t rows, int K, int64_t N, Epilogue ep, int cus);
// Rows per launch of the MFMA kernel for K in-features and N out-features,
// or 0 when the shape is beyond its 32-bit buffer offsets: the packed weights
// must stay below 2^31 bytes, N at most 2^24, and a launch covers a slice of
// rows (a multiple of 256, at least 256) whose q and output stay below 2^31
// bytes each.
inline int64_t gemm_row_slice(int64_t K, int64_t N) {
  if (K <= 0 || N <= 0) return 0;
  if ((K / 16) * N * 4 >= (int64_t(1) << 31) || N > (int64_t(1) << 24)) return 0;
  const int64_t by_q = ((int64_t(1) << 31) - 1) / K;
  const int64_t by_y = ((int64_t(1) << 31) - 1) / (4 * N);
  const int64_t slice = ((by_q < by_y ? by_q : by_y) / 256) * 256;
  return slice < 256 ? 0 : slice;
}

// Interleave the packed gate and up projections of a GLU, [K/16][L] each,
// into [K/16][2L] blocks of 16 columns (gate, up, gate, ...); L % 16 == 0.
// MLGRU recurrence over B sequences of T tokens, fcg [B*T][3d] (forget gate,
// candidate, output gate), d % 4 == 0:
//   h_t = f_t h_{t-1} + (1 - f_t) c_t,  o'_t = g_t sigmoid(h_t).
// The sequence is cut into chunks of `chunk` tokens; with more than one
// chunk `ws` holds mlgru_scan_ws_floats(B, T, d) floats (chunk summaries and
// carries), else it is unused.  h0 may be null (h_0 = 0) and may alias h_last.
int64_t mlgru_chunk_len(int64_t B, int64_t T, int64_t d);
int64_t mlgru_scan_ws_floats(int64_t B, int64_t T, int64_t d);
hipError_t launch_mlgru_scan(const float* fcg, const float* h0, float* o, float* h_last, int64_t B,
                             int64_t T, int64_t d, float* ws, hipStream_t stream);

// ---- backward (bwd.hip: final sums; bwd_gemm.hip: the two products) ----
// out[c] = sum over p < nparts of partials[p * cols + c] (fp64, fixed order).
hipError_t launch_col_final(const double* partials, int64_t nparts, int64_t cols, float* out, hipStream_t stream);
// out[i] = sum over s < S of parts[s * n + i], in order, in fp64.
hipError_t launch_sum_parts(const float* parts, int64_t S, int64_t n, float* out, hipStream_t stream);

// Codes re-packed n-major: Wn [ceil(Np/16)][K] (bwd_nmajor_words(N, K)
// words with Np = N rounded up to 8), codes of n >= N set to t = 0.
int64_t bwd_nmajor_words(int64_t N, int64_t K);
hipError_t launch_pack_nmajor(const uint32_t* Wpacked, int64_t N, int64_t Np, int K, uint32_t* Wn,
                              hipStream_t stream);
// dst [M][N8] = src [M][N] with zero columns N .. N8 - 1.
hipError_t launch_pad_rows(const uint16_t* src, int64_t M, int64_t N, int64_t N8, uint16_t* dst,
                           hipStream_t stream);
// dY kernel: dO [M][Np] bf16 (Np % 8 == 0) against Wn; writes rg = r gamma dY
// into rg [M][K], s_part [bwd_dy_col_tiles(K)][M] and (if not null) dg_part
// [bwd_dy_row_tiles(M)][K] and db_part [bwd_dy_row_tiles(M)][N] (the column
// sums of dO per row tile, for db).  bwd_dy_row_slice(Np, K) == 0: shape not
// supported (32-bit offsets).
int64_t bwd_dy_col_tiles(int64_t K);
int64_t bwd_dy_row_tiles(int64_t M);
int64_t bwd_dy_row_slice(int64_t Np, int64_t K);
hipError_t launch_dy(const uint16_t* dO, int64_t M, int64_t N, int64_t Np, const uint32_t* Wn,
                     const float* w_scale, const void* x, bool x_is_f32, const float* gamma, const float* rstd,
                     int K, float* rg, double* s_part, double* dg_part, double* db_part, hipStream_t stream);
// dx = rg - (r^3 s / K) x in place; dgamma from the row-tile partials.
hipError_t launch_dx_finish(float* dx, const void* x, bool x_is_f32, const float* rstd, const double* s_part,
                            int64_t M, int K, hipStream_t stream);
hipError_t launch_dgamma_finish(const double* dg_part, int64_t M, int K, float* dgamma, hipStream_t stream);
// db[n] = sum over the row tiles of db_part (fp64, tile order).
hipError_t launch_db_finish(const double* db_part, int64_t M, int64_t N, float* db, hipStream_t stream);
// Work units of the dW kernel.  split_all > 1: every tile's token range is
// split into split_all parts, written to out [split_all][N][K] and added by
// launch_sum_parts.  Otherwise tiles [0, full) are whole units and the
// stages (64 tokens each) of the tail_tiles tiles after them, laid end to
// end, go to tail_units units of tail_steps stages; their pieces land in
// bwd_dw_parts_bytes of slots that launch_dw adds into out by a second
// kernel.  N * K * 4 must stay below 2^31.
struct DwPlan {
  int64_t tiles = 0, split_all = 1, full = 0, tail_tiles = 0, tail_steps = 0, tail_units = 0;
};
constexpr int64_t kDwMinTailSteps = 8;
DwPlan bwd_dw_plan(int64_t M, int64_t N, int64_t K, int64_t Np, int cus);
size_t bwd_dw_parts_bytes(const DwPlan& plan);
hipError_t launch_dw(const uint16_t* dO, const int8_t* q, const float* a_scale, int64_t M, int64_t Np, int64_t N,
                     int K, float* out, float* parts, const DwPlan& plan, hipStream_t stream);

hipError_t launch_glu_pack(const uint32_t* Wg, const uint32_t* Wu, int64_t L, int K, uint32_t* Wgu,
                           hipStream_t stream);

}  // namespace mmf
