// The two products of the BitLinear backward (Algorithm 1, backward_pass;
// the straight-through estimator of Sec. "Surrogate Gradient" passes the
// gradient through both quantisers) on the gfx950 matrix cores, with bf16
// operands and fp32 accumulation (v_mfma_f32_16x16x32_bf16):
//
//   dY = dO Wt^T   contraction over the N output features.  The weight
//                  operand is read as 2-bit codes and expanded in registers
//                  into exact bf16 values; the RMSNorm backward's row-wise
//                  pieces run in the epilogue (rms_norm_bwd).
//   dW = dO^T Yq   contraction over the M tokens.  Both operands are read
//                  column-wise, through the LDS transpose reads of gfx950;
//                  Yq = bf16(q a_scale) is formed from the int8 activations
//                  while they are staged into LDS.
//
// dY kernel.  The codes are re-packed once per call "n-major": word (jn, k)
// holds the codes c = t + 1 of t[16 jn + e][k] for e = 0 .. 15, so the 8
// contraction values one MFMA lane needs (8 consecutive n of one column k)
// are 16 bits of one word.  Within the word, e = 8h + 2d + p (half h, pair
// d, parity p) sits at bit 8 (1 - h) + 2d + 16p: a rotation by 24 h bits
// brings the lane's half to bits 8 .. 15 and 24 .. 31, after which one AND-OR
// per pair makes a byte-permute selector [zero, c_2d, zero, c_2d+1] and one
// v_perm_b32 against the table {0xBF, 0x00, 0x3F} turns it into the bf16
// pair (t_2d / 2, t_2d+1 / 2) -- the value +-0.5 has a zero low byte, +-1
// would not.  The sum is doubled (exactly) in the epilogue.
//
// The dY tile is 128 tokens x 512 input features; 8 waves each own 128 x 64
// (8 x 4 MFMA tiles), so each expanded code fragment feeds eight MFMAs.  The
// stage pipeline (3-slot LDS ring, LDS-DMA copies issued one per fragment
// group, one k64-byte step ahead) is the one of the prefill contraction: the
// dO rows are 128-byte slices of 64 bf16 values, exactly as the int8 rows of
// q are 128 int8 values there.
//
// Epilogue of dY (each value produced once, from registers):
//   dY = fp32((2 w_scale) acc),  g = gamma dY,  rg = r g  -> stored to dx
//   s_part[tile k][m]   = sum over the tile's columns of g x    (fp64)
//   dg_part[tile m][k]  = sum over the tile's rows of dY x r    (fp64)
// dx = rg - (r^3 s / K) x is finished by a streaming pass once every column
// tile of the row has its s_part (dx_finish_kernel).
//
// dW kernel.  Tile 256 output features (n) x 256 input features (k), 8 waves
// of 128 x 64; the contraction runs over stages of 64 tokens in a 2-slot LDS
// ring (64 KB each): the dO slice [64][256] bf16 arrives by LDS-DMA, the q
// slice [64][256] int8 through registers, where it becomes bf16(q a_scale)
// (q + 128 converted from its unsigned byte, then fma(q + 128, a, -128 a):
// the product q a rounded once, as the fp32 product is) before it is written
// to LDS.  Operand fragments (8 consecutive tokens of one column per lane)
// come from ds_read_b64_tr_b16: within each group of 16 lanes, lane j + 4e
// names the 4 columns c0 + 4j .. + 3 of token row e, and lane L receives
// column c0 + L of the four rows.  The 512-byte LDS rows are chunk-swizzled
// (16-byte chunk c in slot c ^ sw(row), sw(row) = 2 (4 (row & 1) | ((row >> 1)
// & 1) | 2 ((row >> 3) & 1))) so the rows one transpose read spans fall on
// distinct bank groups, and so do the Yq stores of two consecutive rows.
// When the output has few tiles the token range is split, and the parts are
// added in fp64 in a fixed order; otherwise the tiles past the last whole
// round of workgroups have their stages spread evenly over one more round of
// units (each covering the end of one tile and the start of the next at
// most), whose pieces a second kernel adds in token order.  The pieces meet
// only through the kernel boundary: a last-arriver sum inside the kernel
// needs a device-scope release per piece, which writes back the L2 and
// measured slower than running those tiles unsplit.
#include "gemm_common.h"
#include "mmf_device.h"
#include "mmf_launch.h"

namespace mmf {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef short v4s __attribute__((ext_vector_type(4)));

constexpr int kBlock = 256;

// ---------------------------------------------------------------------------
// n-major re-pack of the codes: Wn [ceil(N/16)][K] from Wpacked [K/16][N]
// (word (j, n): code of k = 16j + 4i + b at bit 8b + 2i); n >= N gets code 1.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int nmajor_bit(int e) { return 8 * (1 - (e >> 3)) + 2 * ((e >> 1) & 3) + 16 * (e & 1); }

// Workgroup (x: jn, y: 256 columns k0 .. k0 + 255): the 16 x 16 input words of
// rows k0 / 16 .. + 15 and columns n = 16 jn .. + 15 go through LDS, then
// thread k assembles output word (jn, k0 + k) from the 16 words of its row.
__global__ __launch_bounds__(kBlock) void pack_nmajor_kernel(const uint32_t* __restrict__ Wp, int64_t N, int K,
                                                             int64_t JN, uint32_t* __restrict__ Wn) {
  __shared__ uint32_t tile[16][17];
  const int t = threadIdx.x;
  const int64_t jn = blockIdx.x;
  const int k0 = blockIdx.y * kBlock;
  {
    const int j = t >> 4, e = t & 15;  // input word (k0 / 16 + j, 16 jn + e)
    const int64_t n = 16 * jn + e;
    const int jr = k0 / 16 + j;
    tile[j][e] = (n < N && jr < K / 16) ? Wp[static_cast<int64_t>(jr) * N + n] : 0x55555555u;  // code 1 = zero
  }
  __syncthreads();
  const int k = k0 + t;
  if (k >= K) return;
  const int sh = 8 * (k & 3) + 2 * ((k >> 2) & 3);
  uint32_t w = 0;
#pragma unroll
  for (int e = 0; e < 16; ++e) w |= ((tile[t >> 4][e] >> sh) & 3u) << nmajor_bit(e);
  Wn[jn * K + k] = w;
}

// dO rows padded with zeros to a multiple of 8 columns (16-byte chunks).
__global__ __launch_bounds__(kBlock) void pad_rows_kernel(const uint16_t* __restrict__ src, int64_t M, int64_t N,
                                                          int64_t N8, uint16_t* __restrict__ dst) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (idx >= M * N8) return;
  const int64_t m = idx / N8, n = idx % N8;
  dst[idx] = n < N ? src[m * N + n] : uint16_t(0);
}

// ---------------------------------------------------------------------------
// dY = dO Wt^T with the RMSNorm-backward epilogue
// ---------------------------------------------------------------------------
namespace dyk {
constexpr int BM = 128, BN = 512, WN = 64, BK = 128, S = 3;
constexpr int kWaves = BN / WN;                        // 8, each over all BM rows
constexpr int kThreads = kWaves * kWave;
constexpr int FM = BM / 16, FN = WN / 16;              // 8 x 4 MFMA tiles per wave
constexpr int KS = BK / 64;                            // 32-value steps per stage (64 bytes each)
constexpr int kABytes = BM * BK;
constexpr int kAInstr = kABytes / 1024;
constexpr int kRowsPerInstr = 1024 / BK;
constexpr int kWordRows = BK / 32;                     // 64 n per stage = 4 n-major word rows
constexpr int kBRow = BN + 16;                         // padded word row
constexpr int kBBytes = kWordRows * kBRow * 4;
constexpr int kBInstr = kWordRows * BN / 256;
constexpr int kAPerWave = kAInstr / kWaves, kBPerWave = kBInstr / kWaves;
constexpr int kLoadsPerStage = kAPerWave + kBPerWave;
constexpr int kStageBytes = kABytes + kBBytes;
static_assert(kAInstr % kWaves == 0 && kBInstr % kWaves == 0, "loads must split evenly");
static_assert(kLoadsPerStage <= FM, "one stage load per fragment group");
static_assert(FN == 4 && FM >= 2 * FN, "expansion schedule: four words, one per late fragment");
static_assert(S * kStageBytes >= kWaves * 4 * BM * 8, "row-sum reduction reuses the ring");
constexpr int kDbRedBytes = kWaves * kWave * 8;        // per-wave fp64 scratch of the db column sums
static_assert(BK == 128 && kWaves == 8 && BM == 128, "db duty: wave w sums chunk w of every row");
}  // namespace dyk

// Expanded code fragment of one lane: 8 bf16 values t / 2 (see the file head).
__device__ __forceinline__ v4i expand_bf16_half(uint32_t w, uint32_t rot) {
  const uint32_t x = __builtin_amdgcn_alignbit(w, w, rot);
  v4i r;
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const uint32_t sel = ((x >> (2 * d)) & 0x03000300u) | 0x000C000Cu;
    r[d] = static_cast<int>(__builtin_amdgcn_perm(0u, 0x003F00BFu, sel));
  }
  return r;
}

__device__ __forceinline__ v4f mfma_bf16(v4i a, v4i b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a), __builtin_bit_cast(v8bf, b), c, 0,
                                                 0, 0);
}

template <typename XT> struct X4;
template <> struct X4<uint16_t> {
  static __device__ void load(const uint16_t* p, float* f) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    f[0] = __uint_as_float(v.x << 16);
    f[1] = __uint_as_float(v.x & 0xFFFF0000u);
    f[2] = __uint_as_float(v.y << 16);
    f[3] = __uint_as_float(v.y & 0xFFFF0000u);
  }
};
template <> struct X4<float> {
  static __device__ void load(const float* p, float* f) {
    const float4 v = *reinterpret_cast<const float4*>(p);
    f[0] = v.x; f[1] = v.y; f[2] = v.z; f[3] = v.w;
  }
};

// dO [M][Np] bf16 (Np % 8 == 0, zero columns past N), Wn [ceil(Np/16)][K].
// rg [M][K] (the dx buffer), s_part [ceil(K/BN)][ld_s] (row m at column m),
// dg_part [ceil(M/BM)][K] or null, db_part [ceil(M/BM)][N] or null.
//
// db duty: the column tiles of a row tile read the same dO rows, so each
// 64-column stage of dO is summed over the row tile's 128 rows by one of them
// (stage kt by column tile kt % ntn) while the stage is in LDS: wave w sums
// the 8 columns of chunk w, lane (row group g8 = lane / 8, column lane % 8)
// the 16 rows g8 + 8 i in fp64 (bf16 values are exact in fp64), then the 8
// row groups are added in order through the wave's own LDS scratch and the
// sum goes to db_part[tm][n].
template <typename XT>
__global__ __launch_bounds__(dyk::kThreads) void dy_kernel(
    const uint16_t* __restrict__ dO, const uint32_t* __restrict__ Wn, const float* __restrict__ w_scale,
    const XT* __restrict__ x, const float* __restrict__ gamma, const float* __restrict__ rstd,
    float* __restrict__ rg, double* __restrict__ s_part, int64_t ld_s, double* __restrict__ dg_part,
    double* __restrict__ db_part, int M, int N, int Np, int K) {
  using namespace dyk;
  __shared__ __attribute__((aligned(16))) char smem[S * kStageBytes + kDbRedBytes];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wn = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15;
  const int g = lane >> 4;
  int64_t tm, tn;
  tile_coords(blockIdx.x, (M + BM - 1) / BM, (K + BN - 1) / BN, tm, tn);
  const int m0 = static_cast<int>(tm) * BM;
  const int k0 = static_cast<int>(tn) * BN;
  const int rowb = 2 * Np;                      // bytes per dO row
  const int JN = (Np + 15) / 16;
  const int KT = (rowb + BK - 1) / BK;

  // A (dO rows): as the prefill contraction's q rows, 128 bytes per stage
  uint32_t a_src[kAPerWave];
  int a_chunk[kAPerWave];
#pragma unroll
  for (int i = 0; i < kAPerWave; ++i) {
    const int r = (wn * kAPerWave + i) * kRowsPerInstr + lane / 8;
    const int c = (lane % 8) ^ a_swz(r);
    a_chunk[i] = c * 16;
    a_src[i] = static_cast<uint32_t>(m0 + r) * static_cast<uint32_t>(rowb) + static_cast<uint32_t>(c * 16);
  }
  // B (n-major words): instruction = word row jj of the stage, 256 columns
  const int b_jj = wn / (BN / 256), b_q = wn % (BN / 256);
  const int b_dst = b_jj * kBRow * 4 + b_q * 1024;
  const uint32_t b_src = 4u * (static_cast<uint32_t>(b_jj) * static_cast<uint32_t>(K) +
                               static_cast<uint32_t>(k0 + b_q * 256 + 4 * lane));
  const uint32_t b_row = 4u * static_cast<uint32_t>(K);
  const v4i adesc = buffer_desc(dO, static_cast<uint32_t>(M) * static_cast<uint32_t>(rowb));
  const v4i bdesc = buffer_desc(Wn, static_cast<uint32_t>(JN) * b_row);
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(smem));

  auto issue_one = [&](int kt, int i) {
    const uint32_t base = lds0 + static_cast<uint32_t>((kt % S) * kStageBytes);
    const int kb = kt * BK;
    if (i < kAPerWave) {
      const uint32_t off = (kb + a_chunk[i] < rowb) ? a_src[i] + static_cast<uint32_t>(kb) : kOutOfRange;
      lds_dma16(__builtin_amdgcn_readfirstlane(base + (wn * kAPerWave + i) * 1024), off, adesc);
    } else {
      const int j0 = kt * kWordRows;
      const uint32_t off = (j0 + b_jj < JN) ? b_src + static_cast<uint32_t>(j0) * b_row : kOutOfRange;
      lds_dma16(__builtin_amdgcn_readfirstlane(base + kABytes + b_dst), off, bdesc);
    }
  };

  v4f acc[FM][FN];
#pragma unroll
  for (int a = 0; a < FM; ++a)
#pragma unroll
    for (int b = 0; b < FN; ++b) acc[a][b] = v4f{0.f, 0.f, 0.f, 0.f};

  v4i af[FM];
  uint32_t bw[FN];
  v4i be[2][FN];
  const uint32_t rot = (g & 1) ? 24u : 0u;
  auto a_read = [&](int s, int fm) -> v4i {
    const int kt = s / KS, ks = s % KS;
    const char* st = smem + (kt % S) * kStageBytes;
    const int row = fm * 16 + l16;
    const int c = (ks * 4 + g) ^ a_swz(row);
    return *reinterpret_cast<const v4i*>(st + row * BK + c * 16);
  };
  auto b_read = [&](int s, int f) -> uint32_t {
    const int kt = s / KS, ks = s % KS;
    const uint32_t* Bs = reinterpret_cast<const uint32_t*>(smem + (kt % S) * kStageBytes + kABytes);
    return Bs[(ks * 2 + (g >> 1)) * kBRow + wn * WN + f * 16 + l16];
  };

#pragma unroll
  for (int p = 0; p < S - 1; ++p)
#pragma unroll
    for (int i = 0; i < kLoadsPerStage; ++i) issue_one(p, i);
  __builtin_amdgcn_s_waitcnt(MMF_WAIT_VM((S - 2) * kLoadsPerStage));
  __builtin_amdgcn_s_barrier();
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) af[fm] = a_read(0, fm);
#pragma unroll
  for (int f = 0; f < FN; ++f) bw[f] = b_read(0, f);
#pragma unroll
  for (int f = 0; f < FN; ++f) be[0][f] = expand_bf16_half(bw[f], rot);

  // db duty of stage kt (see above); its slot stays intact until the barrier
  // of stage kt + 1's last step, and every read here is consumed before it
  const int ntn = (K + BN - 1) / BN;
  double* db_red = reinterpret_cast<double*>(smem + S * kStageBytes) + wn * kWave;
  auto db_stage = [&](int kt) {
    const char* st = smem + (kt % S) * kStageBytes;
    const int dc = lane & 7, g8 = lane >> 3;
    double sum = 0.0;
#pragma unroll
    for (int i = 0; i < BM / 8; ++i) {
      const int r = g8 + 8 * i;
      const uint32_t v = *reinterpret_cast<const uint16_t*>(st + r * BK + ((wn ^ a_swz(r)) << 4) + 2 * dc);
      sum += static_cast<double>(__uint_as_float(v << 16));
    }
    db_red[lane] = sum;
    if (lane < 8) {
      double t = 0.0;
#pragma unroll
      for (int j = 0; j < 8; ++j) t += db_red[8 * j + lane];
      const int n = kt * (BK / 2) + wn * 8 + lane;
      if (n < N) db_part[tm * N + n] = t;
    }
  };

  // one 32-value step s: its MFMAs, the fragment reads of step s + 1 and
  // the expansion of its words; the last step of a stage waits for the next
  // stage's loads and passes a barrier, then refills the retired slot (and,
  // on its db duty, sums the stage's columns)
  auto step = [&](int s, v4i (&bc)[FN], v4i (&bn)[FN]) {
    const int kt = s / KS, ks = s % KS;
    const bool refill = (ks == KS - 1);
    __builtin_amdgcn_sched_barrier(0);
    if (refill) {
      __builtin_amdgcn_s_waitcnt(MMF_WAIT_VM((S - 3) * kLoadsPerStage));
      __builtin_amdgcn_s_barrier();
    }
#pragma unroll
    for (int f = 0; f < FN; ++f) bw[f] = b_read(s + 1, f);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
#pragma unroll
      for (int f = 0; f < FN; ++f) acc[fm][f] = mfma_bf16(bc[f], af[fm], acc[fm][f]);
      af[fm] = a_read(s + 1, fm);
      if (refill && fm < kLoadsPerStage) issue_one(kt + S - 1, fm);
      if (fm >= FM - FN) bn[fm - (FM - FN)] = expand_bf16_half(bw[fm - (FM - FN)], rot);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (refill && db_part != nullptr && kt % ntn == tn) db_stage(kt);
  };
  const int steps = KT * KS;
  int s = 0;
  for (; s + 1 < steps; s += 2) {
    step(s, be[0], be[1]);
    step(s + 1, be[1], be[0]);
  }
  if (s < steps) step(s, be[0], be[1]);
  __builtin_amdgcn_s_waitcnt(MMF_WAIT_VM_LGKM0(0));
  __syncthreads();  // the ring is reused below

  // ---- epilogue: lane (g, l16) holds row l16 and columns 4g .. 4g + 3 of
  // each 16 x 16 block (the MFMA took the codes as its first operand) ----
  const float w2 = 2.0f * w_scale[0];
  float gam[FN][4];
#pragma unroll
  for (int f = 0; f < FN; ++f) {
    const int k = k0 + wn * WN + f * 16 + 4 * g;
#pragma unroll
    for (int e = 0; e < 4; ++e) gam[f][e] = (gamma != nullptr && k < K) ? gamma[k + e] : 1.0f;
  }
  double dgp[FN][4];
#pragma unroll
  for (int f = 0; f < FN; ++f)
#pragma unroll
    for (int e = 0; e < 4; ++e) dgp[f][e] = 0.0;
  double* red = reinterpret_cast<double*>(smem);  // [kWaves][4][BM]
  // r g leaves through a private LDS buffer per wave after the row sums'
  // region, 16 rows at a time: written as the lane holds it (row l16, four
  // columns of each 16-column block), read back as four store instructions
  // of 4 rows x 256 contiguous bytes (one wave's LDS operations complete in
  // issue order, so no barrier and one buffer for every row group)
  constexpr int kRgRow = WN * 4 + 16;
  static_assert(kWaves * 4 * BM * 8 + kWaves * 16 * kRgRow <= S * kStageBytes, "row sums and staging fit the ring");
  char* const sbuf = smem + kWaves * 4 * BM * 8 + wn * 16 * kRgRow;
  const int rr = lane >> 4, qq = lane & 15;
  const int kq = k0 + wn * WN + 4 * qq;  // read-back lane's four columns
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    const int lr = fm * 16 + l16;
    const int m = m0 + lr;
    const bool row_ok = m < M;
    const float r = row_ok ? rstd[m] : 0.0f;
    const double rd = static_cast<double>(r);
    double sp = 0.0;
#pragma unroll
    for (int f = 0; f < FN; ++f) {
      const int k = k0 + wn * WN + f * 16 + 4 * g;
      float o[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      if (row_ok && k < K) {
        float xv[4];
        X4<XT>::load(x + static_cast<int64_t>(m) * K + k, xv);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float dy = w2 * acc[fm][f][e];
          const float gk = gam[f][e] * dy;
          o[e] = r * gk;
          sp += static_cast<double>(gk) * static_cast<double>(xv[e]);
          dgp[f][e] += static_cast<double>(dy) * static_cast<double>(xv[e]) * rd;
        }
      }
      *reinterpret_cast<float4*>(sbuf + l16 * kRgRow + (f * 16 + 4 * g) * 4) = make_float4(o[0], o[1], o[2], o[3]);
    }
    red[(wn * 4 + g) * BM + lr] = sp;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
    __builtin_amdgcn_s_waitcnt(MMF_WAIT_LGKM0);
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 4 * i + rr;
      const float4 v = *reinterpret_cast<const float4*>(sbuf + row * kRgRow + qq * 16);
      const int mr = m0 + fm * 16 + row;
      if (mr < M && kq < K) *reinterpret_cast<float4*>(rg + static_cast<int64_t>(mr) * K + kq) = v;
    }
  }
  if (dg_part != nullptr) {
#pragma unroll
    for (int f = 0; f < FN; ++f) {
      const int k = k0 + wn * WN + f * 16 + 4 * g;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        double v = dgp[f][e];
        v += dpp_f64<kDppXor1>(v);
        v += dpp_f64<kDppXor2>(v);
        v += dpp_f64<kDppHalfMirror>(v);
        v += dpp_f64<kDppMirror>(v);
        if (l16 == 0 && k < K) dg_part[tm * K + k + e] = v;
      }
    }
  }
  __syncthreads();
  if (tid < BM && m0 + tid < M) {
    double sum = 0.0;
    for (int w = 0; w < kWaves; ++w)
#pragma unroll
      for (int gg = 0; gg < 4; ++gg) sum += red[(w * 4 + gg) * BM + tid];
    s_part[tn * ld_s + m0 + tid] = sum;
  }
}

// dx = rg - coef x, coef = r^3 s / K with s the fp64 sum of the row's column
// tile partials (in tile order); four values per thread.
template <typename XT>
__global__ __launch_bounds__(kBlock) void dx_finish_kernel(float* __restrict__ dx, const XT* __restrict__ x,
                                                           const float* __restrict__ rstd,
                                                           const double* __restrict__ s_part, int nkt,
                                                           int64_t M, int K) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  const int64_t e0 = idx * 4;
  if (e0 >= M * K) return;
  const int64_t m = e0 / K;
  double s = 0.0;
  for (int t = 0; t < nkt; ++t) s += s_part[t * M + m];
  const double rd = static_cast<double>(rstd[m]);
  const float coef = static_cast<float>(rd * rd * rd * s / static_cast<double>(K));
  float xv[4];
  X4<XT>::load(x + e0, xv);
  const float4 v = *reinterpret_cast<const float4*>(dx + e0);
  *reinterpret_cast<float4*>(dx + e0) = make_float4(v.x - coef * xv[0], v.y - coef * xv[1],
                                                    v.z - coef * xv[2], v.w - coef * xv[3]);
}

// ---------------------------------------------------------------------------
// dW = dO^T Yq
// ---------------------------------------------------------------------------
namespace dwk {
constexpr int BN = 256, BK = 256, WN = 128, WK = 64, BT = 64, S = 2;
constexpr int kWavesK = BK / WK;                       // 4
constexpr int kWaves = (BN / WN) * kWavesK;            // 8
constexpr int kThreads = kWaves * kWave;
constexpr int FM = WN / 16, FN = WK / 16;              // 8 x 4 MFMA tiles per wave
constexpr int KS = BT / 32;                            // 32-token steps per stage
constexpr int kRow = 512;                              // bytes per LDS row (256 bf16)
constexpr int kTile = BT * kRow;                       // 32 KB
constexpr int kStageBytes = 2 * kTile;                 // dO slice, then Yq slice
constexpr int kDmaPerWave = kTile / 1024 / kWaves;     // 4 LDS-DMA instructions per wave per stage
constexpr int kQPerThread = BT * BK / kThreads;        // 32 int8 of one token row
static_assert(kQPerThread == 32, "q staging: four 8-byte loads per thread");
static_assert(S == 2 && KS == 2, "stage schedule below");
}  // namespace dwk

// Row swizzle of the dW kernel's 512-byte LDS rows (see the file head).
__device__ __forceinline__ int dw_swz(int row) {
  return 2 * (((row & 1) << 2) | ((row >> 1) & 1) | (((row >> 3) & 1) << 1));
}

// q (int8, 8 values) -> bf16(q a): one 16-byte LDS chunk, 4 dwords.
typedef float v2f __attribute__((ext_vector_type(2)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v2f{lo, hi}, v2bf));
}
__device__ __forceinline__ void yq8(int2 qv, float a, uint32_t* out) {
  const float am = -128.0f * a;
  const int w[2] = {qv.x, qv.y};
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const uint32_t u = static_cast<uint32_t>(w[i]) ^ 0x80808080u;  // q + 128 as unsigned bytes
    const float f0 = __builtin_fmaf(static_cast<float>(u & 0xFFu), a, am);
    const float f1 = __builtin_fmaf(static_cast<float>((u >> 8) & 0xFFu), a, am);
    const float f2 = __builtin_fmaf(static_cast<float>((u >> 16) & 0xFFu), a, am);
    const float f3 = __builtin_fmaf(static_cast<float>(u >> 24), a, am);
    out[2 * i] = bf16x2(f0, f1);
    out[2 * i + 1] = bf16x2(f2, f3);
  }
}

// Output offset (bytes) of element 4 g of 16 x 16 block (fm, f) held by
// thread tid of tile (n0, k0) in out [N][K], or kOutOfRange past N or K:
// lane (g, l16) of wave (wn, wk) holds output feature n = l16 and input
// features 4g .. 4g + 3 of each block (Yq was the MFMAs' first operand).
__device__ __forceinline__ uint32_t dw_out_off(int n0, int k0, int tid, int fm, int f, int N, int K) {
  using namespace dwk;
  const int wave = tid >> 6, lane = tid & 63;
  const int n = n0 + (wave / kWavesK) * WN + fm * 16 + (lane & 15);
  const int k = k0 + (wave % kWavesK) * WK + f * 16 + 4 * (lane >> 4);
  return (n < N && k < K) ? (static_cast<uint32_t>(n) * static_cast<uint32_t>(K) + static_cast<uint32_t>(k)) * 4u
                          : kOutOfRange;
}

// dO [T][Np] and q [T][K] of T tokens; out [N][K], or [split_all][N][K]
// parts when split_all > 1; parts: the tail pieces' slots (see DwPlan).
__global__ __launch_bounds__(dwk::kThreads) void dw_kernel(const uint16_t* __restrict__ dO,
                                                           const int8_t* __restrict__ q,
                                                           const float* __restrict__ a_scale, int T, int Np,
                                                           int N, int K, DwPlan plan, float* __restrict__ out_base,
                                                           float* __restrict__ parts) {
  using namespace dwk;
  __shared__ __attribute__((aligned(16))) char smem[S * kStageBytes];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave / kWavesK, wk = wave % kWavesK;
  const int l16 = lane & 15;
  const int g = lane >> 4;
  // work unit -> one or two pieces (tile, token range [ta, tb), slot; slot
  // -1: stored to out)
  const int u = blockIdx.x;
  int npiece = 1, tile_a, ta_a, tb_a, slot_a = -1, tile_b = 0, ta_b = 0, tb_b = 0, slot_b = -1;
  float* out = out_base;
  if (plan.split_all > 1) {
    const int split = static_cast<int>(u / plan.tiles);
    const int nsplit = static_cast<int>(plan.split_all);
    const int per = (T + nsplit - 1) / nsplit;
    const int per64 = (per + BT - 1) / BT * BT;
    tile_a = static_cast<int>(u % plan.tiles);
    ta_a = split * per64 < T ? split * per64 : T;
    tb_a = ta_a + per64 < T ? ta_a + per64 : T;
    out = out_base + static_cast<int64_t>(split) * N * K;
  } else if (u < plan.full) {
    tile_a = u;
    ta_a = 0;
    tb_a = T;
  } else {
    // tail unit v: stages [v I, v I + I) of the tail tiles' stages laid end
    // to end (I = tail_steps <= a tile's stage count, so at most two tiles)
    const int64_t kts = (T + BT - 1) / BT;
    const int64_t v = u - plan.full;
    const int64_t a = v * plan.tail_steps;
    const int64_t b = a + plan.tail_steps < plan.tail_tiles * kts ? a + plan.tail_steps : plan.tail_tiles * kts;
    const int64_t ia = a / kts, ib = (b - 1) / kts;
    tile_a = static_cast<int>(plan.full + ia);
    ta_a = static_cast<int>((a - ia * kts) * BT);
    tb_a = static_cast<int>(((ia == ib ? b : (ia + 1) * kts) - ia * kts) * BT);
    tb_a = tb_a < T ? tb_a : T;
    slot_a = static_cast<int>(v + ia);
    if (ib != ia) {
      npiece = 2;
      tile_b = static_cast<int>(plan.full + ib);
      tb_b = static_cast<int>((b - ib * kts) * BT);
      tb_b = tb_b < T ? tb_b : T;
      slot_b = static_cast<int>(v + ib);
    }
  }
  for (int pc = 0; pc < npiece; ++pc) {
    const int tile = pc ? tile_b : tile_a;
    const int t0 = pc ? ta_b : ta_a, t1 = pc ? tb_b : tb_a;
    const int slot = pc ? slot_b : slot_a;
    if (pc) {
      // the first piece's LDS reads and stores are done everywhere before the
      // second's copies go out
      __builtin_amdgcn_s_waitcnt(MMF_WAIT_VM_LGKM0(0));
      __builtin_amdgcn_s_barrier();
    }
    int64_t tnn, tkk;
    tile_coords(tile, (N + BN - 1) / BN, (K + BK - 1) / BK, tnn, tkk);
    const int n0 = static_cast<int>(tnn) * BN;
    const int k0 = static_cast<int>(tkk) * BK;
    const int KT = t1 > t0 ? (t1 - t0 + BT - 1) / BT : 0;
    const uint32_t rowb = 2u * static_cast<uint32_t>(Np);
    const v4i ddesc = buffer_desc(dO + static_cast<int64_t>(t0) * Np, static_cast<uint32_t>(t1 - t0) * rowb);
    const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(smem));

    // dO DMA: instruction i of the stage covers token rows 2i, 2i + 1; lane
    // (row half, slot) copies logical chunk slot ^ sw(row)
    uint32_t d_src[kDmaPerWave];
#pragma unroll
    for (int i = 0; i < kDmaPerWave; ++i) {
      const int ins = wave * kDmaPerWave + i;
      const int row = 2 * ins + (lane >> 5);
      const int c = (lane & 31) ^ dw_swz(row);
      const int n = n0 + c * 8;
      d_src[i] = n < Np ? static_cast<uint32_t>(row) * rowb + 2u * static_cast<uint32_t>(n) : kOutOfRange;
    }
    // q staging: thread (row tid / 8, p = tid % 8) owns the 8-column chunks
    // p + 8i (i = 0 .. 3) of its token row, so the 8 threads of a row write 8
    // distinct bank groups per store and the next row (swizzle differing by
    // 8) the other 8.
    const int q_row = tid >> 3, q_part = tid & 7;
    uint32_t q_src[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int k = k0 + 8 * (q_part + 8 * i);
      q_src[i] = k < K ? static_cast<uint32_t>(q_row) * static_cast<uint32_t>(K) + static_cast<uint32_t>(k)
                       : kOutOfRange;
    }
    const int q_sw = dw_swz(q_row);
    auto issue_dma = [&](int kt) {
      const uint32_t base = lds0 + static_cast<uint32_t>((kt % S) * kStageBytes);
      const uint32_t tb = static_cast<uint32_t>(kt * BT) * rowb;
      const bool live = kt < KT;
#pragma unroll
      for (int i = 0; i < kDmaPerWave; ++i) {
        const uint32_t off = (d_src[i] == kOutOfRange || !live) ? kOutOfRange : d_src[i] + tb;
        lds_dma16(__builtin_amdgcn_readfirstlane(base + (wave * kDmaPerWave + i) * 1024), off, ddesc);
      }
    };
    // The thread's 32 q values and its token's a_scale (zero past the range)
    // are loaded by inline assembly, so the compiler inserts no wait for them
    // (its count of outstanding loads would not include the LDS-DMA copies
    // issued behind them, and it would wait for those too); wait_q ties the
    // registers to an explicit vmcnt wait.  Every load is issued and consumed
    // within one loop iteration, so the registers never pass a loop back-edge.
    const v4i qdesc =
        buffer_desc(q + static_cast<int64_t>(t0) * K, static_cast<uint32_t>(t1 - t0) * static_cast<uint32_t>(K));
    const v4i adesc = buffer_desc(a_scale + t0, static_cast<uint32_t>(t1 - t0) * 4u);
    int2 qv0, qv1, qv2, qv3;
    float qa;
    auto issue_q = [&](int kt) {
      const uint32_t tb = static_cast<uint32_t>(kt * BT) * static_cast<uint32_t>(K);
      const bool live = kt < KT;
      uint32_t o[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = (q_src[i] == kOutOfRange || !live) ? kOutOfRange : q_src[i] + tb;
      const uint32_t oa = live ? 4u * static_cast<uint32_t>(kt * BT + q_row) : kOutOfRange;
      asm volatile("buffer_load_dwordx2 %0, %1, %2, 0 offen" : "=v"(qv0) : "v"(o[0]), "s"(qdesc) : "memory");
      asm volatile("buffer_load_dwordx2 %0, %1, %2, 0 offen" : "=v"(qv1) : "v"(o[1]), "s"(qdesc) : "memory");
      asm volatile("buffer_load_dwordx2 %0, %1, %2, 0 offen" : "=v"(qv2) : "v"(o[2]), "s"(qdesc) : "memory");
      asm volatile("buffer_load_dwordx2 %0, %1, %2, 0 offen" : "=v"(qv3) : "v"(o[3]), "s"(qdesc) : "memory");
      asm volatile("buffer_load_dword %0, %1, %2, 0 offen" : "=v"(qa) : "v"(oa), "s"(adesc) : "memory");
    };
    // wait until only the kDmaPerWave copies issued behind the q loads remain
    auto wait_q = [&]() {
      asm volatile("s_waitcnt vmcnt(%5)"
                   : "+v"(qv0), "+v"(qv1), "+v"(qv2), "+v"(qv3), "+v"(qa)
                   : "n"(kDmaPerWave)
                   : "memory");
    };
    // the Yq of chunk i of this thread's token row (quarter i of its q)
    auto write_yq_chunk = [&](int kt, int i) {
      char* dst = smem + (kt % S) * kStageBytes + kTile + q_row * kRow;
      const int2 qi = i == 0 ? qv0 : i == 1 ? qv1 : i == 2 ? qv2 : qv3;
      uint32_t b[4];
      yq8(qi, qa, b);
      const int slot = (q_part + 8 * i) ^ q_sw;
      *reinterpret_cast<v4i*>(dst + slot * 16) =
          v4i{static_cast<int>(b[0]), static_cast<int>(b[1]), static_cast<int>(b[2]), static_cast<int>(b[3])};
    };
    auto write_yq = [&](int kt) {
#pragma unroll
      for (int i = 0; i < 4; ++i) write_yq_chunk(kt, i);
    };

    // transpose-read offsets: lane (g, l16) names token row 8g + 4h + (l16 >> 2)
    // and columns c0 + 4 (l16 & 3) .. + 3
    const int tj = l16 & 3, te = l16 >> 2;
    const int r_sw = dw_swz(8 * g + te);  // the same for both halves and steps
    auto tr_off = [&](int c0) -> uint32_t {
      const int chunk = (c0 >> 3) + (tj >> 1);
      return static_cast<uint32_t>(((chunk ^ r_sw) << 4) + 8 * (tj & 1));
    };
    uint32_t offA[FM], offB[FN];
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) offA[fm] = tr_off(wn * WN + fm * 16);
#pragma unroll
    for (int f = 0; f < FN; ++f) offB[f] = kTile + tr_off(wk * WK + f * 16);
    const uint32_t row_base = static_cast<uint32_t>((8 * g + te) * kRow);
    auto frag = [&](int s, uint32_t off) -> v4i {
      const int kt = s / KS, ks = s % KS;
      const char* base = smem + (kt % S) * kStageBytes + ks * 32 * kRow + row_base + off;
      typedef __attribute__((address_space(3))) v4s lds_v4s;
      const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(base));
      const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(base + 4 * kRow));
      const int2 l2 = __builtin_bit_cast(int2, lo), h2 = __builtin_bit_cast(int2, hi);
      return v4i{l2.x, l2.y, h2.x, h2.y};
    };

    v4f acc[FM][FN];
#pragma unroll
    for (int a = 0; a < FM; ++a)
#pragma unroll
      for (int b = 0; b < FN; ++b) acc[a][b] = v4f{0.f, 0.f, 0.f, 0.f};

    // Schedule (stage kt = steps 2kt, 2kt + 1; slot kt % 2).  Step 2kt turns
    // stage kt + 1's q into Yq in the other slot; the first thing of step
    // 2kt + 1 is the barrier that makes stage kt + 1 complete everywhere, after
    // which stage kt + 2's q and dO copies go out (into the slot of stage kt,
    // whose last reads were the read-ahead of step 2kt) and step 2kt + 1's
    // MFMAs run with the read-ahead of step 2kt + 2.  Copies past the last
    // stage read zero and are never used.  After the prologue's copies of
    // stage 1 only those are waited for (vmcnt kDmaPerWave), which also
    // covers stage 0's copies and q loads issued before them.
    if (KT > 0) {
      v4i af[FM], b0[FN], b1[FN];
      // one 32-token step: its MFMAs, with the next step's fragments read and
      // (convert) a quarter of a stage's Yq formed behind every other group
      auto mma = [&](const v4i (&bc)[FN], v4i (&bn)[FN], int next_step, bool read_next, bool convert, int conv_kt) {
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int fm = 0; fm < FM; ++fm) {
#pragma unroll
          for (int f = 0; f < FN; ++f) acc[fm][f] = mfma_bf16(bc[f], af[fm], acc[fm][f]);
          if (read_next) af[fm] = frag(next_step, offA[fm]);
          if (read_next && fm < FN) bn[fm] = frag(next_step, offB[fm]);
          if (convert && fm == 1) wait_q();
          if (convert && (fm & 1)) write_yq_chunk(conv_kt, fm >> 1);
          __builtin_amdgcn_sched_barrier(0);
        }
      };
      issue_q(0);
      issue_dma(0);
      wait_q();
      write_yq(0);
      const bool two = KT > 1;
      if (two) issue_q(1);
      issue_dma(1);
      __builtin_amdgcn_s_waitcnt(MMF_WAIT_VM_LGKM0(kDmaPerWave));
      __builtin_amdgcn_s_barrier();
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) af[fm] = frag(0, offA[fm]);
#pragma unroll
      for (int f = 0; f < FN; ++f) b0[f] = frag(0, offB[f]);
      // step 0: stage 1's Yq, MFMAs with the read-ahead of step 1
      mma(b0, b1, 1, true, two, 1);
      for (int kt = 0; kt < KT; ++kt) {
        const bool next = kt + 1 < KT;
        // step 2kt + 1
        __builtin_amdgcn_s_waitcnt(MMF_WAIT_VM_LGKM0(0));
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        // (q is loaded exactly when step 2kt + 2 converts it, under the same
        // condition, so its registers stay live until their wait)
        const bool q_next = kt + 2 < KT;
        if (q_next) issue_q(kt + 2);
        issue_dma(kt + 2);
        mma(b1, b0, 2 * kt + 2, next, false, 0);
        // step 2kt + 2 (the first step of stage kt + 1): stage kt + 2's Yq
        if (next) mma(b0, b1, 2 * kt + 3, true, q_next, kt + 2);
      }
      __builtin_amdgcn_s_waitcnt(MMF_WAIT_VM_LGKM0(0));
    }

    if (slot >= 0) {
      // a tail piece: its sums to the slot in register order, thread-minor
      float* dst = parts + static_cast<int64_t>(slot) * (BN * BK) + 4 * tid;
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int f = 0; f < FN; ++f) *reinterpret_cast<v4f*>(dst + (fm * FN + f) * (4 * kThreads)) = acc[fm][f];
    } else {
      // the tile leaves through a private LDS buffer per wave in the ring
      // (every wave is past the ring's last stage after the barrier), 16
      // output features at a time: written as the lane holds them (feature
      // l16, four input features of each 16-wide block), read back as four
      // store instructions of 4 features x 256 contiguous bytes (one wave's
      // LDS operations complete in issue order: no further barrier)
      constexpr int kRow = WK * 4 + 16;
      static_assert(kWaves * 16 * kRow <= S * kStageBytes, "the staging buffers fit the ring");
      __builtin_amdgcn_s_barrier();
      char* const sbuf = smem + wave * 16 * kRow;
      const uint32_t out_bytes = static_cast<uint32_t>(N) * static_cast<uint32_t>(K) * 4u;
      const __amdgpu_buffer_rsrc_t orsrc =
          __builtin_amdgcn_make_buffer_rsrc(out, 0, static_cast<int>(out_bytes), kBufferFlags);
      const int rr = lane >> 4, qq = lane & 15;
      const int kq = k0 + wk * WK + 4 * qq;
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) {
#pragma unroll
        for (int f = 0; f < FN; ++f)
          *reinterpret_cast<v4f*>(sbuf + l16 * kRow + (f * 16 + 4 * g) * 4) = acc[fm][f];
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
        __builtin_amdgcn_s_waitcnt(MMF_WAIT_LGKM0);
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const v4i v = *reinterpret_cast<const v4i*>(sbuf + (4 * i + rr) * kRow + qq * 16);
          const int n = n0 + wn * WN + fm * 16 + 4 * i + rr;
          const uint32_t off = (n < N && kq < K)
                                   ? (static_cast<uint32_t>(n) * static_cast<uint32_t>(K) + static_cast<uint32_t>(kq)) * 4u
                                   : kOutOfRange;
          __builtin_amdgcn_raw_buffer_store_b128(v, orsrc, off, 0, 0);
        }
      }
    }
  }
}

// The tail tiles of a DwPlan: blocks ti * kFixupSplit + j add blocks e of
// tile full + ti held in registers e = j E .. j E + E - 1 (E = FM FN /
// kFixupSplit), over the tile's pieces in token order (the units overlapping
// its stages, slot = unit + ti), and store them like the kernel's epilogue.
constexpr int kFixupSplit = 8;
static_assert(dwk::FM * dwk::FN % kFixupSplit == 0, "fixup blocks take whole register groups");
__global__ __launch_bounds__(dwk::kThreads) void dw_fixup_kernel(const float* __restrict__ parts, int T, int N,
                                                                 int K, DwPlan plan, float* __restrict__ out) {
  using namespace dwk;
  constexpr int E = FM * FN / kFixupSplit;
  const int tid = threadIdx.x;
  const int64_t ti = blockIdx.x / kFixupSplit;
  const int e0 = static_cast<int>(blockIdx.x % kFixupSplit) * E;
  const int64_t kts = (T + BT - 1) / BT;
  const int64_t v0 = ti * kts / plan.tail_steps, v1 = ((ti + 1) * kts - 1) / plan.tail_steps;
  int64_t tnn, tkk;
  tile_coords(plan.full + ti, (N + BN - 1) / BN, (K + BK - 1) / BK, tnn, tkk);
  const int n0 = static_cast<int>(tnn) * BN;
  const int k0 = static_cast<int>(tkk) * BK;
  const float* src = parts + (v0 + ti) * (BN * BK) + 4 * tid;
  v4f sum[E];
#pragma unroll
  for (int i = 0; i < E; ++i) sum[i] = *reinterpret_cast<const v4f*>(src + (e0 + i) * (4 * kThreads));
  for (int64_t v = v0 + 1; v <= v1; ++v) {
    const float* p = src + (v - v0) * (BN * BK);
#pragma unroll
    for (int i = 0; i < E; ++i) sum[i] += *reinterpret_cast<const v4f*>(p + (e0 + i) * (4 * kThreads));
  }
  const uint32_t out_bytes = static_cast<uint32_t>(N) * static_cast<uint32_t>(K) * 4u;
  const __amdgpu_buffer_rsrc_t orsrc =
      __builtin_amdgcn_make_buffer_rsrc(out, 0, static_cast<int>(out_bytes), kBufferFlags);
#pragma unroll
  for (int i = 0; i < E; ++i)
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4i, sum[i]), orsrc,
                                           dw_out_off(n0, k0, tid, (e0 + i) / FN, (e0 + i) % FN, N, K), 0, 0);
}

}  // namespace

// ---- launchers ----

int64_t bwd_nmajor_words(int64_t N, int64_t K) { return ((N + 7) / 8 * 8 + 15) / 16 * K; }

hipError_t launch_pack_nmajor(const uint32_t* Wpacked, int64_t N, int64_t Np, int K, uint32_t* Wn,
                              hipStream_t stream) {
  const int64_t JN = (Np + 15) / 16;
  if (JN * K == 0) return hipSuccess;
  hipLaunchKernelGGL(pack_nmajor_kernel, dim3(static_cast<unsigned>(JN), static_cast<unsigned>((K + kBlock - 1) / kBlock)),
                     dim3(kBlock), 0, stream, Wpacked, N, K, JN, Wn);
  return hipGetLastError();
}

hipError_t launch_pad_rows(const uint16_t* src, int64_t M, int64_t N, int64_t N8, uint16_t* dst, hipStream_t stream) {
  const int64_t total = M * N8;
  if (total == 0) return hipSuccess;
  hipLaunchKernelGGL(pad_rows_kernel, dim3(static_cast<unsigned>((total + kBlock - 1) / kBlock)), dim3(kBlock), 0,
                     stream, src, M, N, N8, dst);
  return hipGetLastError();
}

int64_t bwd_dy_col_tiles(int64_t K) { return (K + dyk::BN - 1) / dyk::BN; }
int64_t bwd_dy_row_tiles(int64_t M) { return (M + dyk::BM - 1) / dyk::BM; }

int64_t bwd_dy_row_slice(int64_t Np, int64_t K) {
  // 32-bit buffer offsets: dO rows (2 Np bytes each) and n-major words of
  // one launch stay below 2^31 bytes; slices are whole row tiles
  const int64_t lim = (int64_t(1) << 31) - 1;
  if (((Np + 15) / 16) * K * 4 > lim) return 0;
  int64_t rows = lim / (2 * Np);
  rows = rows / dyk::BM * dyk::BM;
  return rows;
}

hipError_t launch_dy(const uint16_t* dO, int64_t M, int64_t N, int64_t Np, const uint32_t* Wn,
                     const float* w_scale, const void* x, bool x_is_f32, const float* gamma, const float* rstd,
                     int K, float* rg, double* s_part, double* dg_part, double* db_part, hipStream_t stream) {
  const int64_t slice = bwd_dy_row_slice(Np, K);
  if (slice == 0) return hipErrorInvalidValue;
  for (int64_t mb = 0; mb < M; mb += slice) {
    const int64_t rows = M - mb < slice ? M - mb : slice;
    const dim3 grid(static_cast<unsigned>(bwd_dy_row_tiles(rows) * bwd_dy_col_tiles(K)));
    double* dgp = dg_part ? dg_part + (mb / dyk::BM) * K : nullptr;
    double* dbp = db_part ? db_part + (mb / dyk::BM) * N : nullptr;
    if (x_is_f32)
      hipLaunchKernelGGL(dy_kernel<float>, grid, dim3(dyk::kThreads), 0, stream, dO + mb * Np, Wn, w_scale,
                         static_cast<const float*>(x) + mb * K, gamma, rstd + mb, rg + mb * K, s_part + mb, M,
                         dgp, dbp, static_cast<int>(rows), static_cast<int>(N), static_cast<int>(Np), K);
    else
      hipLaunchKernelGGL(dy_kernel<uint16_t>, grid, dim3(dyk::kThreads), 0, stream, dO + mb * Np, Wn, w_scale,
                         static_cast<const uint16_t*>(x) + mb * K, gamma, rstd + mb, rg + mb * K, s_part + mb, M,
                         dgp, dbp, static_cast<int>(rows), static_cast<int>(N), static_cast<int>(Np), K);
  }
  return hipGetLastError();
}

hipError_t launch_dx_finish(float* dx, const void* x, bool x_is_f32, const float* rstd, const double* s_part,
                            int64_t M, int K, hipStream_t stream) {
  const int64_t total = M * K / 4;
  if (total == 0) return hipSuccess;
  const int nkt = static_cast<int>(bwd_dy_col_tiles(K));
  const dim3 grid(static_cast<unsigned>((total + kBlock - 1) / kBlock));
  if (x_is_f32)
    hipLaunchKernelGGL(dx_finish_kernel<float>, grid, dim3(kBlock), 0, stream, dx, static_cast<const float*>(x), rstd,
                       s_part, nkt, M, K);
  else
    hipLaunchKernelGGL(dx_finish_kernel<uint16_t>, grid, dim3(kBlock), 0, stream, dx,
                       static_cast<const uint16_t*>(x), rstd, s_part, nkt, M, K);
  return hipGetLastError();
}

hipError_t launch_dgamma_finish(const double* dg_part, int64_t M, int K, float* dgamma, hipStream_t stream) {
  return launch_col_final(dg_part, bwd_dy_row_tiles(M), K, dgamma, stream);
}

hipError_t launch_db_finish(const double* db_part, int64_t M, int64_t N, float* db, hipStream_t stream) {
  return launch_col_final(db_part, bwd_dy_row_tiles(M), N, db, stream);
}

DwPlan bwd_dw_plan(int64_t M, int64_t N, int64_t K, int64_t Np, int cus) {
  DwPlan p;
  p.tiles = ((N + dwk::BN - 1) / dwk::BN) * ((K + dwk::BK - 1) / dwk::BK);
  p.full = p.tiles;
  const int64_t lim = (int64_t(1) << 31) - 1;
  // 32-bit offsets: a part's rows, rounded up to whole stages, plus one
  // stage of rows past its end (which read as zero) stay below 2^31 bytes of
  // dO and of q
  auto fits = [&](int64_t s) {
    const int64_t rows = (M + s - 1) / s + 2 * dwk::BT;
    return rows * 2 * Np <= lim && rows * K <= lim;
  };
  const int64_t kts = (M + dwk::BT - 1) / dwk::BT;
  if (p.tiles * 2 > cus && fits(1)) {
    // whole tiles in full rounds; the last, partial round's stages spread
    // over up to `cus` units of at least kDwMinTailSteps stages, when that
    // saves an eighth of a tile's time or more
    const int64_t r = p.tiles % cus;
    if (r > 0 && kts > 0) {
      int64_t steps = (r * kts + cus - 1) / cus;
      if (steps < kDwMinTailSteps) steps = kDwMinTailSteps;
      if (8 * steps <= 7 * kts) {
        p.full = p.tiles - r;
        p.tail_tiles = r;
        p.tail_steps = steps;
        p.tail_units = (r * kts + steps - 1) / steps;
      }
    }
    return p;
  }
  // few tiles: split every tile's tokens while parts keep 512 tokens
  int64_t S = 1;
  while (p.tiles * S < (cus * 3) / 4 && M / (2 * S) >= 512) S *= 2;
  while (!fits(S)) S *= 2;
  p.split_all = S;
  return p;
}

size_t bwd_dw_parts_bytes(const DwPlan& p) {
  return p.tail_units > 0 ? static_cast<size_t>(p.tail_units + p.tail_tiles) * dwk::BN * dwk::BK * sizeof(float) : 0;
}

hipError_t launch_dw(const uint16_t* dO, const int8_t* q, const float* a_scale, int64_t M, int64_t Np, int64_t N,
                     int K, float* out, float* parts, const DwPlan& plan, hipStream_t stream) {
  if (N * K * 4 > (int64_t(1) << 31) - 1) return hipErrorInvalidValue;
  if (plan.tail_units > 0 && parts == nullptr) return hipErrorInvalidValue;
  const int64_t units = plan.split_all > 1 ? plan.tiles * plan.split_all : plan.full + plan.tail_units;
  if (units == 0) return hipSuccess;
  hipLaunchKernelGGL(dw_kernel, dim3(static_cast<unsigned>(units)), dim3(dwk::kThreads), 0, stream, dO, q, a_scale,
                     static_cast<int>(M), static_cast<int>(Np), static_cast<int>(N), K, plan, out, parts);
  if (plan.tail_units > 0)
    hipLaunchKernelGGL(dw_fixup_kernel, dim3(static_cast<unsigned>(plan.tail_tiles * kFixupSplit)), dim3(dwk::kThreads),
                       0, stream,
                       parts, static_cast<int>(M), static_cast<int>(N), K, plan, out);
  return hipGetLastError();
}

}  // namespace mmf
