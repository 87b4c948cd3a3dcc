// Fused decode forward (1 to 16 tokens): RMSNorm + absmax int8 quantisation +
// ternary accumulation + dequantisation in one launch.  Included by the
// decode_*.hip files, one per activation source, which compile in parallel.
//
// Each workgroup owns C = 16 F output columns over the whole K dimension of
// the [K/16][N] packed weights.  A "step" is 4 word rows (64 k values) of the
// workgroup's columns; lane (g, l16) of a wave reads word row 4 s + g of the
// F consecutive columns F l16 .. F l16 + F - 1 with one 4-, 8- or 16-byte
// load (256-byte strips of the column block per word row), and the 16 waves
// split the steps into contiguous ranges.
//
// Latency is what limits a decode launch, so every load is issued at entry:
// first the activations (x and gamma, or the pre-quantised q), then every
// weight load of the wave.  The RMSNorm and quantisation of the token rows
// into LDS then run while the weights stream in; the barriers between their
// phases wait for LDS only (fences of the local address space), never for the
// weight loads in flight.  The contraction consumes the weight loads in issue
// order, each as soon as it has landed.
//
// The contraction: v_mfma_i32_16x16x64_i8 over the codes c = t + 1, 16
// columns by the 16 token rows of q (rows past the token count read as zero),
// for one token as for sixteen.  The epilogue subtracts sum_k q, giving the
// ternary sum of the paper (+q where t = 1, -q where t = -1, nothing where
// t = 0), and dequantises.
#pragma once
#include "mmf_device.h"
#include "mmf_launch.h"

namespace mmf {
namespace dec {

constexpr int kWaves = 16;
constexpr int kThreads = kWaves * kWave;  // 1024
constexpr int kMaxTokens = kDecodeMaxTokens;
constexpr int kMaxRowWaves = 4;            // waves that normalise one token row
// column sums of token m at red[m * kRedStride + column]: the odd stride puts
// the same column of different tokens on different LDS banks
constexpr int kRedStride = kWave + 1;
constexpr int kLdsDmaChunk = 1024;         // bytes of q one LDS-DMA wave instruction copies
constexpr int kMaxQChunks = (kDecodeMaxLdsQ / kLdsDmaChunk + kWaves - 1) / kWaves;  // per wave
constexpr int kBufferFlags = 0x00020000;   // gfx9 buffer descriptor word 3
constexpr uint32_t kOutOfRange = 0x80000000u;  // past every buffer (each < 2^31 bytes)
typedef int v4i __attribute__((ext_vector_type(4)));

// kMlgru: the activations are the MLGRU's output gate o' = g sigmoid(f h +
// (1 - f) c), formed on load from the gates fcg [M][3K] and the state h [M][K]
// (fp32); workgroup 0 also stores the new state.
enum class Src { kBf16, kF32, kQuantised, kMlgru };

template <Src S>
constexpr int vec_elems() { return (S == Src::kF32 || S == Src::kMlgru) ? 4 : 8; }

// Token rows are normalised and quantised by groups of G waves, G = 4 for up
// to 4 tokens, 2 for up to 8, 1 for up to 16; group r owns row r and the
// remaining waves do no row work.  At most one wave per SIMD works on a row:
// the per-row steps (reductions, the fp64 root) are latency chains, and more
// waves on a SIMD would only serialise the same instructions.  G is a
// compile-time parameter of the kernel (index arithmetic with a run-time
// group size measured 0.4-0.5 us slower per one-token launch).
constexpr int row_waves_for(int mt) { return mt <= 4 ? 4 : mt <= 8 ? 2 : 1; }

// Barrier for LDS traffic only: the fences are restricted to the local
// address space, so the barrier waits for this wave's LDS operations but not
// for its global loads in flight (a plain __syncthreads would wait for them).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

struct Shared {
  int8_t* q;        // [mt][q_stride]
  int q_stride;     // bytes from one token row of q to the next
  int* red;         // [kMaxTokens][kRedStride] column sums (LDS atomics)
  double* slot_d;   // [kWaves]
  float* slot_f;    // [kWaves]
  int* slot_i;      // [kWaves]
  float* a_scale;   // [kMaxTokens]
  int* rowsum;      // [kMaxTokens]
};

constexpr int kScalarBytes = sizeof(int) * kMaxTokens * kRedStride +
                             (sizeof(double) + sizeof(float) + sizeof(int)) * kWaves +
                             (sizeof(float) + sizeof(int)) * kMaxTokens;

__device__ __forceinline__ Shared carve(char* base, int q_bytes, int q_stride) {
  Shared s;
  s.q = reinterpret_cast<int8_t*>(base);
  s.q_stride = q_stride;
  char* p = base + q_bytes;
  s.red = reinterpret_cast<int*>(p);
  p += sizeof(int) * kMaxTokens * kRedStride;
  s.slot_d = reinterpret_cast<double*>(p);
  p += sizeof(double) * kWaves;
  s.slot_f = reinterpret_cast<float*>(p);
  p += sizeof(float) * kWaves;
  s.slot_i = reinterpret_cast<int*>(p);
  p += sizeof(int) * kWaves;
  s.a_scale = reinterpret_cast<float*>(p);
  p += sizeof(float) * kMaxTokens;
  s.rowsum = reinterpret_cast<int*>(p);
  return s;
}

// Activation staging for the fused path: the raw x and gamma vectors of this
// thread (VP 16-byte vectors of its row), loaded at entry and left untouched
// until begin(), so that the weight loads issued after them are not held up.
template <int G, Src S, int VP>
struct RowStage {
  static constexpr int E = vec_elems<S>();
  static constexpr int VM = S == Src::kMlgru ? VP : 1;
  uint4 xr[VP];
  uint4 xc[VM], xg[VM], xh[VM];  // kMlgru: c, g and h beside f in xr
  float4 gr[VP][E / 4];
  float f[VP][E];
  int row, gtid, nvec;
  bool active;
  float* h_out;

  __device__ __forceinline__ void load(const void* xv, const float* __restrict__ gamma, int K, int mt,
                                       const float* h_in, float* h_store) {
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    row = wave / G;
    gtid = threadIdx.x - row * G * kWave;
    active = row < mt;  // wave-uniform; waves past mt * G do no row work
    nvec = K / E;
    h_out = h_store;
    if (!active) return;
    if constexpr (S == Src::kMlgru) {
      // f, c, g of the row side by side in fcg; h through a buffer resource
      // of size 0 when there is no state (reads as h = 0)
      const float* fr = static_cast<const float*>(xv) + static_cast<int64_t>(row) * 3 * K;
      const __amdgpu_buffer_rsrc_t frsrc = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<float*>(fr), 0, 3 * K * 4, kBufferFlags);
      const __amdgpu_buffer_rsrc_t hrsrc = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<float*>(h_in), 0, h_in != nullptr ? mt * K * 4 : 0, kBufferFlags);
#pragma unroll
      for (int p = 0; p < VP; ++p) {
        const int v = gtid + G * kWave * p;
        const uint32_t off = v < nvec ? static_cast<uint32_t>(v * 16) : kOutOfRange;
        xr[p] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(frsrc, off, 0, 0));
        xc[p] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(frsrc, off, K * 4, 0));
        xg[p] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(frsrc, off, 2 * K * 4, 0));
        xh[p] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                              hrsrc, v < nvec ? static_cast<uint32_t>((row * K + v * E) * 4)
                                                              : kOutOfRange, 0, 0));
      }
    } else {
      // the row through a buffer resource of its own K elements: vectors
      // past its end read as zero, so the values need no mask
      const __amdgpu_buffer_rsrc_t xrsrc = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<char*>(static_cast<const char*>(xv) + static_cast<int64_t>(row) * K * (16 / E)), 0,
          K * (16 / E), kBufferFlags);
#pragma unroll
      for (int p = 0; p < VP; ++p) {
        const int v = gtid + G * kWave * p;
        xr[p] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                              xrsrc, static_cast<uint32_t>(v * 16), 0, 0));
      }
    }
    // gamma through a buffer resource of size 0 when it is NULL: the loads
    // return zeros without touching memory and need no branch
    const __amdgpu_buffer_rsrc_t grsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(gamma), 0, gamma != nullptr ? K * 4 : 0, kBufferFlags);
#pragma unroll
    for (int p = 0; p < VP; ++p) {
      const int v = gtid + G * kWave * p;
#pragma unroll
      for (int e4 = 0; e4 < E / 4; ++e4) {
        const uint32_t off = v < nvec ? static_cast<uint32_t>((v * E + 4 * e4) * 4) : kOutOfRange;
        gr[p][e4] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(grsrc, off, 0, 0));
      }
    }
  }

  // values of vector p as fp32 (zero outside the row)
  __device__ __forceinline__ void values(int p, float* out) const {
    const int v = gtid + G * kWave * p;
    const bool ok = v < nvec;
    if constexpr (S == Src::kMlgru) {
      const float fv[4] = {__uint_as_float(xr[p].x), __uint_as_float(xr[p].y), __uint_as_float(xr[p].z),
                           __uint_as_float(xr[p].w)};
      const float cv[4] = {__uint_as_float(xc[p].x), __uint_as_float(xc[p].y), __uint_as_float(xc[p].z),
                           __uint_as_float(xc[p].w)};
      const float gv[4] = {__uint_as_float(xg[p].x), __uint_as_float(xg[p].y), __uint_as_float(xg[p].z),
                           __uint_as_float(xg[p].w)};
      const float hv[4] = {__uint_as_float(xh[p].x), __uint_as_float(xh[p].y), __uint_as_float(xh[p].z),
                           __uint_as_float(xh[p].w)};
      float hn[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        hn[e] = mlgru_step(hv[e], fv[e], cv[e]);
        out[e] = ok ? mlgru_out_gate(gv[e], hn[e]) : 0.0f;
      }
      // the new state, once per call: workgroup 0 stores it
      if (ok && h_out != nullptr && blockIdx.x == 0)
        *reinterpret_cast<float4*>(h_out + static_cast<int64_t>(row) * (nvec * 4) + v * 4) =
            make_float4(hn[0], hn[1], hn[2], hn[3]);
    } else if constexpr (E == 8) {  // zero past the row's end (see load)
      const uint32_t w[4] = {xr[p].x, xr[p].y, xr[p].z, xr[p].w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        out[2 * i] = __uint_as_float(w[i] << 16);
        out[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
      }
    } else {
      out[0] = __uint_as_float(xr[p].x);
      out[1] = __uint_as_float(xr[p].y);
      out[2] = __uint_as_float(xr[p].z);
      out[3] = __uint_as_float(xr[p].w);
    }
  }
  __device__ __forceinline__ float gamma_at(int p, int e) const {
    const float4 g = gr[p][e / 4];
    const int k = e % 4;
    return k == 0 ? g.x : k == 1 ? g.y : k == 2 ? g.z : g.w;
  }

  // RMSNorm, absmax and quantisation of the staged values into LDS, in three
  // phases that the caller separates by LDS barriers, which every wave
  // reaches, while only the waves of a row group do the work (`active` is
  // uniform across a wave).  The row sum of q is left in the per-wave slots.
  // phase 1: this wave's share of the row's sum of squares (where a row wave
  // first waits for its activations)
  __device__ __forceinline__ void sum_squares(const Shared& sh) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (active) {
#pragma unroll
      for (int p = 0; p < VP; ++p) values(p, f[p]);
      double ss = 0.0;
#pragma unroll
      for (int p = 0; p < VP; ++p)
#pragma unroll
        for (int e = 0; e < E; ++e) ss = sum_sq(ss, f[p][e]);
      ss = wave_sum_f64(ss);
      if (lane == 0) sh.slot_d[wave] = ss;
    }
  }
  // phase 2: rstd, the normalised values and this wave's absmax
  __device__ __forceinline__ void scale_absmax(bool has_gamma, int K, const Shared& sh) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int w0 = row * G;
    if (active) {
      double tot = 0.0;
      for (int w = 0; w < G; ++w) tot += sh.slot_d[w0 + w];
      const float r = rms_rstd(tot, K);
      float amax = 0.0f;
#pragma unroll
      for (int p = 0; p < VP; ++p)
#pragma unroll
        for (int e = 0; e < E; ++e) {
          float y = f[p][e] * r;
          if (has_gamma) y = y * gamma_at(p, e);
          f[p][e] = y;  // zero for vectors outside the row
          amax = fmaxf(amax, fabsf(y));
        }
      amax = wave_max_f32(amax);
      if (lane == 0) sh.slot_f[wave] = amax;
    }
  }
  // phase 3: the row scale, q into LDS, the row sums of q
  __device__ __forceinline__ void quantise(const Shared& sh) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int w0 = row * G;
    if (active) {
      float a = 0.0f;
      for (int w = 0; w < G; ++w) a = fmaxf(a, sh.slot_f[w0 + w]);
      a = fmaxf(a, 1e-5f);
      const float s = 127.0f / a;
      int rs = 0;
#pragma unroll
      for (int p = 0; p < VP; ++p) {
        const int v = gtid + G * kWave * p;
        uint32_t packed[E / 4];
#pragma unroll
        for (int gq = 0; gq < E / 4; ++gq) {
          packed[gq] = quantise4(&f[p][4 * gq], s);
          rs = byte_sum4(packed[gq], rs);
        }
        if (v < nvec) {
          int8_t* dst = sh.q + row * sh.q_stride + v * E;
          if constexpr (E == 8)
            *reinterpret_cast<uint2*>(dst) = make_uint2(packed[0], packed[1]);
          else
            *reinterpret_cast<uint32_t*>(dst) = packed[0];
        }
      }
      rs = wave_sum_i32(rs);
      if (lane == 0) sh.slot_i[wave] = rs;
      if (gtid == 0) sh.a_scale[row] = a / 127.0f;
    }
  }
};

// Pre-quantised activations: q copied into LDS by LDS-DMA (global memory
// straight to LDS, 16 bytes per lane and 1 KB per wave instruction, no
// registers involved; the range check of the buffer resource returns zero
// past the end of q), a_scale and q_rowsum by the first mt threads.
struct QStage {
  float a;
  int rs;
  __device__ __forceinline__ void load(const int8_t* __restrict__ q, const float* __restrict__ a_scale,
                                       const int32_t* __restrict__ q_rowsum, int K, int mt, const Shared& sh) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int bytes = mt * K;
    const int chunks = (bytes + kLdsDmaChunk - 1) / kLdsDmaChunk;
    const uint64_t qa = reinterpret_cast<uint64_t>(q);
    const v4i desc = {static_cast<int>(static_cast<uint32_t>(qa)), static_cast<int>((qa >> 32) & 0xFFFF), bytes,
                      kBufferFlags};
    const uint32_t lds_q = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(sh.q));
    // with padded rows (q_stride > K, only when K % 1024 == 0) a chunk lies
    // inside one row: chunk ch is row ch / cpr, bytes (ch % cpr) KB of it
    const int cpr = sh.q_stride > K ? K / kLdsDmaChunk : 1;
    const int rstride = sh.q_stride > K ? sh.q_stride : kLdsDmaChunk;
#pragma unroll
    for (int i = 0; i < kMaxQChunks; ++i) {
      const int ch = wave + kWaves * i;
      if (ch < chunks) {  // wave-uniform
        const uint32_t off = static_cast<uint32_t>(ch * kLdsDmaChunk + lane * 16);
        const int lds_off = (ch / cpr) * rstride + (ch % cpr) * kLdsDmaChunk;
        const uint32_t dst = __builtin_amdgcn_readfirstlane(lds_q + static_cast<uint32_t>(lds_off));
        asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                     :
                     : "s"(dst), "v"(off), "s"(desc)
                     : "memory", "m0");
      }
    }
    const int t = static_cast<int>(threadIdx.x) < mt ? static_cast<int>(threadIdx.x) : 0;
    a = a_scale != nullptr ? a_scale[t] : 0.0f;
    rs = q_rowsum[t];
  }
  // after the wave's LDS-DMA copies have landed
  __device__ __forceinline__ void store(const Shared& sh, int mt) const {
    const int t = static_cast<int>(threadIdx.x) < mt ? static_cast<int>(threadIdx.x) : 0;
    sh.a_scale[t] = a;
    sh.rowsum[t] = rs;
  }
};

// F consecutive packed words (one 4-, 8- or 16-byte buffer load).
template <int F>
struct Words {
  uint32_t w[F];
};
template <int F>
__device__ __forceinline__ Words<F> load_words(__amdgpu_buffer_rsrc_t rsrc, uint32_t voff, uint32_t soff) {
  Words<F> r;
  if constexpr (F == 1) {
    r.w[0] = __builtin_amdgcn_raw_buffer_load_b32(rsrc, voff, soff, 0);
  } else if constexpr (F == 2) {
    const uint2 v = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(rsrc, voff, soff, 0));
    r.w[0] = v.x;
    r.w[1] = v.y;
  } else {
    static_assert(F == 4, "one, two or four words");
    const uint4 v = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, voff, soff, 0));
    r.w[0] = v.x;
    r.w[1] = v.y;
    r.w[2] = v.z;
    r.w[3] = v.w;
  }
  return r;
}

// Kernel arguments in one block, so that the scalar loads that fetch them are
// issued together at entry.
struct Params {
  const uint32_t* Wp;
  const void* x;
  const float* gamma;
  const int8_t* q;
  const float* a_scale;
  const int32_t* q_rowsum;
  const float* w_scale;
  void* out;
  int64_t N;
  int K;
  int mt;
  int q_bytes;
  int q_stride;
  Affine affine;
  const float* h_in;  // kMlgru
  float* h_out;       // kMlgru
};

// G: waves per token row (4, 2 or 1 for up to 4, 8 or 16 tokens).  VP:
// 16-byte activation vectors per row thread.  F: column blocks of 16 per
// workgroup.  NLD: weight loads (steps) in flight per lane, the wave's whole
// range of steps when it has at most 8 (so that no lane issues a load past
// its range); a wave with more steps refills them NLD at a time.
template <int G, Src S, int VP, int F, int NLD, Epilogue EP>
__global__ __launch_bounds__(kThreads) void decode_kernel(const Params prm) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  static_assert(S != Src::kMlgru || EP == Epilogue::kAffineF32, "the MLGRU prologue feeds the output projection");
  static_assert(EP != Epilogue::kAffineF32 || S != Src::kQuantised, "affine epilogue from x only");
  constexpr int C = 16 * F;  // columns per workgroup
  static_assert(EP != Epilogue::kGluF32 || (C >= 32 && S != Src::kQuantised && S != Src::kMlgru),
                "GLU output: whole gate/up block pairs per workgroup, activations from x");
  const int K = prm.K;
  const int mt = prm.mt;  // 1 <= mt <= 16 / G (at most 16)
  const int64_t N = prm.N;
  const Shared sh = carve(smem, prm.q_bytes, prm.q_stride);
  // read at entry: its latency then overlaps the rest of the kernel
  const float wscale = (EP == Epilogue::kDequantF32 || EP == Epilogue::kGluF32) ? prm.w_scale[0] : 0.0f;
  const float wscale_u = EP == Epilogue::kGluF32 ? prm.w_scale[1] : 0.0f;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, g16 = lane >> 4;
  const int64_t n0 = static_cast<int64_t>(blockIdx.x) * C;
  const int64_t ncol = n0 + F * l16;  // first of this lane's F columns (N % F == 0)
  const int J = K / 16;
  const int steps = (J + 3) / 4;
  const int per_wave = (steps + kWaves - 1) / kWaves;
  const int sb = min(wave * per_wave, steps);
  const int ns = min(sb + per_wave, steps) - sb;  // steps of this wave (uniform)
  // 32-bit offsets: the packed array is < 2^31 bytes (checked by the launcher)
  const __amdgpu_buffer_rsrc_t wrsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(prm.Wp), 0, static_cast<int>(static_cast<uint32_t>(J) * 4u * static_cast<uint32_t>(N)),
      kBufferFlags);
  const uint32_t row_bytes = 4u * static_cast<uint32_t>(N);
  const uint32_t lane_off = static_cast<uint32_t>(g16) * row_bytes + 4u * static_cast<uint32_t>(ncol < N ? ncol : 0);
  const uint32_t step_bytes = 4u * row_bytes;
  // step sb + i of this wave: the lane offset in a VGPR, the step's offset in
  // an SGPR; for i >= ns the lane offset itself lies past the array, so the
  // range check returns zero words (word rows 4 s + g past K/16 of the last
  // step lie past the array too)
  auto load_step = [&](int i) -> Words<F> {
    return load_words<F>(wrsrc, i < ns ? lane_off : kOutOfRange,
                         i < ns ? static_cast<uint32_t>(sb + i) * step_bytes : 0u);
  };

  // 1. activation loads, then every weight load of the first group
  RowStage<G, S == Src::kQuantised ? Src::kBf16 : S, VP> rows;
  QStage qs;
  if constexpr (S == Src::kQuantised) {
    qs.load(prm.q, prm.a_scale, prm.q_rowsum, K, mt, sh);
  } else {
    rows.load(prm.x, prm.gamma, K, mt, prm.h_in, prm.h_out);
  }
  // the factors of the column this thread writes in the affine epilogue
  ColAffine col{};
  if constexpr (EP == Epilogue::kAffineF32) {
    const int64_t cn = n0 + tid % C;
    col = load_col_affine(prm.affine, prm.w_scale, static_cast<uint32_t>(N), cn < N ? static_cast<uint32_t>(cn) : 0u);
  }
  __builtin_amdgcn_sched_barrier(0);
  Words<F> wb[NLD];
  auto issue_weights = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int p = 0; p < NLD; ++p) wb[p] = load_step(p);
    __builtin_amdgcn_sched_barrier(0);
  };

  // 2. the token rows into LDS while the weights stream in.  From x: the
  // weight loads are issued once every row wave has its activations (measured:
  // issued at entry, they delay the activation loads by more than they gain);
  // from a pre-quantised q: at entry, right behind the copies of q.
  for (int i = tid; i < kMaxTokens * kRedStride; i += kThreads) sh.red[i] = 0;
  if constexpr (S == Src::kQuantised) {
    issue_weights();
    // the LDS-DMA copies are this wave's oldest loads: at most NLD (the
    // weights) may still be in flight
    static_assert(NLD <= 15, "vmcnt immediate");
    __builtin_amdgcn_s_waitcnt((NLD & 0xF) | (0x7 << 4) | (0xF << 8));
    qs.store(sh, mt);
  } else {
    rows.sum_squares(sh);
    lds_barrier();
    issue_weights();
    rows.scale_absmax(prm.gamma != nullptr, K, sh);
    lds_barrier();
    rows.quantise(sh);
  }
  lds_barrier();

  // 3. contraction on the matrix cores, each weight load as it lands:
  // 16 x 16 x 64 int8 products of the code bytes of F column blocks (first
  // operand, rows = columns F i + f) against the token rows of q (second
  // operand, rows l16 < mt; the others give zeros).  One token uses one of
  // the 16 operand rows: the products then cost matrix-core cycles, which
  // are otherwise idle, instead of vector-ALU dot products (measured faster
  // for one token as well).  Steps past the wave's range hold zero words
  // (code 0 for every k: they add nothing) and read q at a valid row.
  v4i accf[F];
#pragma unroll
  for (int f = 0; f < F; ++f) accf[f] = v4i{0, 0, 0, 0};
  const bool tok = l16 < mt;
  const int8_t* qrow = sh.q + (tok ? l16 : 0) * sh.q_stride;
  // the steps base .. base + NLD - 1 of this wave from the registers `w`
  // their loads landed in: each is used as soon as its own load is complete
  auto contract = [&](const Words<F>(&w)[NLD], int base) __attribute__((always_inline)) {
#pragma unroll
    for (int p = 0; p < NLD; ++p) {
      const int j = 4 * (sb + base + p) + g16;
      const int jq = j < J ? j : J - 1;
      const uint4 qv = *reinterpret_cast<const uint4*>(qrow + 16 * jq);
      const v4i qf = tok ? __builtin_bit_cast(v4i, qv) : v4i{0, 0, 0, 0};
#pragma unroll
      for (int f = 0; f < F; ++f) {
        const uint32_t x = w[p].w[f];
        const v4i cw = {static_cast<int>(codes4(x, 0)), static_cast<int>(codes4(x, 1)),
                        static_cast<int>(codes4(x, 2)), static_cast<int>(codes4(x, 3))};
        accf[f] = __builtin_amdgcn_mfma_i32_16x16x64_i8(cw, qf, accf[f], 0, 0, 0);
      }
    }
  };
  contract(wb, 0);
  // waves with more than NLD steps (K > 8192): the rest in groups of NLD
  // loads, each group contracted as it lands
  for (int base = NLD; base < ns; base += NLD) {
    Words<F> nb[NLD];
#pragma unroll
    for (int p = 0; p < NLD; ++p) nb[p] = load_step(base + p);
    contract(nb, base);
  }

  // 4. column sums over the waves with LDS integer atomics (exact and
  // order-free): lane (g, l16) holds block f's columns F (4 g + r) + f of
  // token l16; then dequantise
  if (tok) {
#pragma unroll
    for (int f = 0; f < F; ++f)
#pragma unroll
      for (int r = 0; r < 4; ++r) atomicAdd(&sh.red[l16 * kRedStride + F * (4 * g16 + r) + f], accf[f][r]);
  }
  lds_barrier();
  auto row_sum = [&](int m) -> int {
    if constexpr (S == Src::kQuantised) {
      return sh.rowsum[m];
    } else {
      int rsum = 0;
      for (int w = 0; w < G; ++w) rsum += sh.slot_i[m * G + w];
      return rsum;
    }
  };
  if constexpr (EP == Epilogue::kGluF32) {
    // The packed columns alternate 16 gate and 16 up columns, and a
    // workgroup's C columns are C / 32 whole pairs: thread (m, channel) forms
    // SiLU(g) * u of its channel (the formula and order of the MFMA kernel's
    // GLU epilogue, so both give the same bits) into the L = N / 2 wide output.
    constexpr int kHalf = C / 2;
    if (tid < mt * kHalf) {
      const int m = tid / kHalf, hc = tid % kHalf;
      const int cg = (hc / 16) * 32 + hc % 16;  // gate column; up column cg + 16
      const int64_t L = N / 2;
      const int64_t ch = static_cast<int64_t>(blockIdx.x) * kHalf + hc;
      const int rsum = row_sum(m);
      if (ch < L) {
        const float sg = sh.a_scale[m] * wscale, su = sh.a_scale[m] * wscale_u;
        const float gv = static_cast<float>(sh.red[m * kRedStride + cg] - rsum) * sg;
        const float uv = static_cast<float>(sh.red[m * kRedStride + cg + 16] - rsum) * su;
        static_cast<float*>(prm.out)[m * L + ch] = gv * sigmoid_hw(gv) * uv;
      }
    }
  } else if (tid < mt * C) {
    const int m = tid / C, cc = tid % C;
    const int64_t nn = n0 + cc;
    const int rsum = row_sum(m);
    if (nn < N) {
      const int v = sh.red[m * kRedStride + cc] - rsum;
      if constexpr (EP == Epilogue::kDequantF32) {
        static_cast<float*>(prm.out)[m * N + nn] = static_cast<float>(v) * (sh.a_scale[m] * wscale);
      } else if constexpr (EP == Epilogue::kAffineF32) {
        const float z = static_cast<float>(v) * (sh.a_scale[m] * col.ws) + col.bias;
        static_cast<float*>(prm.out)[m * N + nn] = affine_act(z, col.act, col.lb);
      } else {
        static_cast<int32_t*>(prm.out)[m * N + nn] = v;
      }
    }
  }
}

// q row stride in LDS.  The matrix-core contraction reads 16 bytes of one k
// group from each token row at once; rows padded by 16 bytes put those reads
// on distinct banks.  Pre-quantised q is copied in whole 1 KB chunks, so it
// is padded only when a chunk never straddles two rows (K % 1024 == 0).
inline int q_stride_for(bool quantised, int K) {
  return (!quantised || K % kLdsDmaChunk == 0) ? K + 16 : K;
}

// LDS bytes of the q region (whole LDS-DMA chunks)
inline int q_region(int mt, int q_stride) {
  return ((mt * q_stride + kLdsDmaChunk - 1) / kLdsDmaChunk) * kLdsDmaChunk;
}

template <int G, Src S, int VP, int F, int NLD, Epilogue EP>
hipError_t launch_one(const DecodeArgs& a, hipStream_t stream) {
  constexpr int C = 16 * F;
  const int mt = static_cast<int>(a.M);
  const int q_stride = q_stride_for(S == Src::kQuantised, a.K);
  const int region = q_region(mt, q_stride);
  const dim3 grid(static_cast<unsigned>((a.N + C - 1) / C));
  const Params prm{a.Wpacked, a.x, a.gamma, a.q, a.a_scale, a.q_rowsum, a.w_scale, a.out,
                   a.N, a.K, mt, region, q_stride, a.affine, a.h_in, a.h_out};
  hipLaunchKernelGGL((decode_kernel<G, S, VP, F, NLD, EP>), grid, dim3(kThreads), region + kScalarBytes,
                     stream, prm);
  return hipGetLastError();
}

// vectors of 16 bytes per row thread: ceil(K / E / (G * 64))
inline int needed_vp(int mt, int K, bool f32) {
  const int lanes = row_waves_for(mt) * kWave;
  const int nvec = K / (f32 ? 4 : 8);
  return (nvec + lanes - 1) / lanes;
}

// Column blocks per workgroup: as few as keep the grid within one round of
// the 256 CUs (a 1024-thread workgroup fills a CU), with loads aligned to
// their width (N % F == 0); the GLU epilogue needs whole gate/up pairs (F >= 2).
constexpr int kGridRound = 256;
inline int choose_f(int64_t N, bool glu) {
  if (!glu && (N + 15) / 16 <= kGridRound) return 1;
  if (N % 2 == 0 && (N + 31) / 32 <= kGridRound) return 2;
  if (N % 4 == 0) return 4;
  if (N % 2 == 0) return 2;
  return glu ? 0 : 1;
}

// Weight loads in flight per lane: exactly the steps of a wave with the full
// share (1 .. 6 or 8), so that no lane issues loads past its range -- such
// loads return zeros but still cost nearly a real load each (measured: eight
// in flight where five are needed, 7.4 against 6.9 us per d = 5120 decode
// call); beyond 8 steps, 8 at a time.
inline int choose_nld(int K) {
  const int steps = (K / 16 + 3) / 4;
  const int per_wave = (steps + kWaves - 1) / kWaves;
  return per_wave <= 6 ? per_wave : 8;
}

template <int G, Src S, int VP, int F, Epilogue EP>
hipError_t dispatch_nld(const DecodeArgs& a, hipStream_t stream) {
  switch (choose_nld(a.K)) {
    case 1: return launch_one<G, S, VP, F, 1, EP>(a, stream);
    case 2: return launch_one<G, S, VP, F, 2, EP>(a, stream);
    case 3: return launch_one<G, S, VP, F, 3, EP>(a, stream);
    case 4: return launch_one<G, S, VP, F, 4, EP>(a, stream);
    case 5: return launch_one<G, S, VP, F, 5, EP>(a, stream);
    case 6: return launch_one<G, S, VP, F, 6, EP>(a, stream);
    default: return launch_one<G, S, VP, F, 8, EP>(a, stream);
  }
}

template <int G, Src S, int VP, Epilogue EP>
hipError_t dispatch_f(const DecodeArgs& a, hipStream_t stream) {
  const int f = choose_f(a.N, EP == Epilogue::kGluF32);
  if constexpr (EP != Epilogue::kGluF32) {
    if (f == 1) return dispatch_nld<G, S, VP, 1, EP>(a, stream);
  }
  if (f == 2) return dispatch_nld<G, S, VP, 2, EP>(a, stream);
  if (f == 4) return dispatch_nld<G, S, VP, 4, EP>(a, stream);
  return hipErrorInvalidValue;
}

template <int G, Src S, Epilogue EP>
hipError_t dispatch_vp(const DecodeArgs& a, hipStream_t stream) {
  if constexpr (S == Src::kQuantised) {
    return dispatch_f<G, S, 1, EP>(a, stream);
  } else {
    const int vp = needed_vp(static_cast<int>(a.M), a.K, S == Src::kF32 || S == Src::kMlgru);
    if (vp <= 1) return dispatch_f<G, S, 1, EP>(a, stream);
    if (vp <= 2) return dispatch_f<G, S, 2, EP>(a, stream);
    if (vp <= 4) return dispatch_f<G, S, 4, EP>(a, stream);
    return hipErrorInvalidValue;  // excluded by decode_fits
  }
}

template <Src S, Epilogue EP>
hipError_t dispatch(const DecodeArgs& a, hipStream_t stream) {
  switch (row_waves_for(static_cast<int>(a.M))) {
    case 4: return dispatch_vp<4, S, EP>(a, stream);
    case 2: return dispatch_vp<2, S, EP>(a, stream);
    default: return dispatch_vp<1, S, EP>(a, stream);
  }
}

}  // namespace dec

// Per activation source, in decode_<src>.hip.
hipError_t launch_decode_bf16(const DecodeArgs& a, hipStream_t stream);
hipError_t launch_decode_f32(const DecodeArgs& a, hipStream_t stream);
hipError_t launch_decode_q(const DecodeArgs& a, hipStream_t stream);
hipError_t launch_decode_mlgru(const DecodeArgs& a, hipStream_t stream);

}  // namespace mmf
