// Fused decode forward (M <= 8 tokens): RMSNorm + absmax int8 quantisation +
// ternary accumulation + dequantisation in one launch.
//
// Each workgroup owns C = 64/H output columns over the whole K dimension.
// Weight layout [K/16][N] words: for a word row j the lanes of a wave read
// consecutive columns, so each lane owns an output column and accumulates its
// dot products without cross-lane traffic; H lanes share a column by taking
// alternate words and the 16 waves split K into ranges.  The int32 partial
// sums of a column are added in LDS (exact, order-free).
//
// Latency is what limits a decode launch, so the loads are ordered with care:
// memory loads retire in issue order, hence the activation loads (x and gamma,
// or the pre-quantised q) are issued first, then the packed weight words, and
// only then does the kernel wait -- for the activations alone -- and
// normalise/quantise the token rows into LDS while the weights stream in.
// All of these loads are straight-line (clamped addresses, masked values), so
// the compiler can keep them in flight together.
//
// One token: per word of 16 weights, four v_dot4_i32_i8 of the codes
// c = t + 1 against q (one broadcast ds_read_b128).  Two to eight tokens:
// v_mfma_i32_16x16x64_i8 over the same codes, 16 columns by the token rows of
// q (the vector ALU's dot4 rate would fall behind the weight stream at eight
// tokens).  Either way the epilogue subtracts sum_k q, giving the ternary sum
// of the paper (+q where t = 1, -q where t = -1, nothing where t = 0), and
// dequantises.
#include "mmf_device.h"
#include "mmf_launch.h"

namespace mmf {
namespace {

constexpr int kWaves = 16;
constexpr int kThreads = kWaves * kWave;  // 1024
constexpr int kMaxTokens = 8;
constexpr int kMaxRowWaves = 4;           // waves that normalise one token row
// column sums of token m at red[m * kRedStride + column]: the odd stride puts
// the same column of different tokens on different LDS banks
constexpr int kRedStride = kWave + 1;
constexpr int kLdsDmaChunk = 1024;        // bytes of q one LDS-DMA wave instruction copies
constexpr int kMaxQChunks = (kDecodeMaxLdsQ / kLdsDmaChunk + kWaves - 1) / kWaves;  // per wave
constexpr int kWeightDelay = -1;         // < 0: all waves wait for the row waves' x
constexpr int kGridRound = 256;           // workgroups that run at once (one per CU)
constexpr int kMfmaMinTokens = 2;         // token counts contracted on the matrix cores

// kMlgru: the activations are the MLGRU's output gate o' = g sigmoid(f h +
// (1 - f) c), formed on load from the gates fcg [M][3K] and the state h [M][K]
// (fp32); workgroup 0 also stores the new state.
enum class Src { kBf16, kF32, kQuantised, kMlgru };

// Token rows are normalised and quantised by groups of G = min(16 / P, 4)
// waves, P = MT rounded up to a power of two; group g owns row g and the
// remaining waves only stream weights.  At most one wave per SIMD works on a
// row: the per-row steps (reductions, the fp64 root) are latency chains, and
// more waves on a SIMD would only serialise the same instructions.  Each
// thread handles VP 16-byte vectors of its row.
template <int MT>
constexpr int row_groups() { return MT <= 1 ? 1 : MT <= 2 ? 2 : MT <= 4 ? 4 : 8; }
template <int MT>
constexpr int row_waves() {
  return kWaves / row_groups<MT>() < kMaxRowWaves ? kWaves / row_groups<MT>() : kMaxRowWaves;
}
template <Src S>
constexpr int vec_elems() { return (S == Src::kF32 || S == Src::kMlgru) ? 4 : 8; }

struct Shared {
  int8_t* q;        // [MT][q_stride]
  int q_stride;     // bytes from one token row of q to the next
  int* red;         // [kMaxTokens][kRedStride] column sums (LDS atomics)
  double* slot_d;   // [kWaves]
  float* slot_f;    // [kWaves]
  int* slot_i;      // [kWaves]
  float* a_scale;   // [kMaxTokens]
  int* rowsum;      // [kMaxTokens]
};

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

constexpr int kScalarBytes = sizeof(int) * kMaxTokens * kRedStride +
                             (sizeof(double) + sizeof(float) + sizeof(int)) * kWaves +
                             (sizeof(float) + sizeof(int)) * kMaxTokens;

__device__ __forceinline__ void unpack_bf16x8(const uint4& r, float* f) {
  const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}

// Activation staging for the fused path: the raw x and gamma vectors of this
// thread, loaded up front and left untouched until finish(), so that nothing
// waits on them before the weight loads have been issued.
template <int MT, Src S, int VP>
struct RowStage {
  static constexpr int E = vec_elems<S>();
  static constexpr int G = row_waves<MT>();  // waves per row
  static constexpr int VM = S == Src::kMlgru ? VP : 1;
  uint4 xr[VP];
  uint4 xc[VM], xg[VM], xh[VM];  // kMlgru: c, g and h beside f in xr
  float4 gr[VP][E / 4];
  int row, gtid, nvec;
  bool active;
  float* h_out;

  __device__ __forceinline__ void load(const void* xv, const float* __restrict__ gamma, int K, bool inactive_skip = false,
                       const float* h_in = nullptr, float* h_store = nullptr) {
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    row = wave / G;
    gtid = threadIdx.x - row * G * kWave;
    active = row < MT;  // waves past MT * G take no part in the row work
    nvec = K / E;
    h_out = h_store;
    if (inactive_skip && !active) return;  // wave-uniform
    const int srow = active ? row : 0;
    if constexpr (S == Src::kMlgru) {
      // f, c, g of row srow side by side in fcg; h through a buffer resource
      // of size 0 when there is no state (reads as h = 0)
      const float* fr = static_cast<const float*>(xv) + static_cast<int64_t>(srow) * 3 * K;
      const uint4* fv = reinterpret_cast<const uint4*>(fr);
      const uint4* cv = reinterpret_cast<const uint4*>(fr + K);
      const uint4* gv = reinterpret_cast<const uint4*>(fr + 2 * K);
      const __amdgpu_buffer_rsrc_t hrsrc = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<float*>(h_in), 0, h_in != nullptr ? MT * K * 4 : 0, 0x00020000);
#pragma unroll
      for (int p = 0; p < VP; ++p) {
        const int v = gtid + G * kWave * p;
        const int sv = (active && v < nvec) ? v : 0;
        xr[p] = fv[sv];
        xc[p] = cv[sv];
        xg[p] = gv[sv];
        xh[p] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                              hrsrc, static_cast<uint32_t>((srow * K + sv * E) * 4), 0, 0));
      }
    } else {
      // the row through a buffer resource of its own K elements (size 0 for
      // a wave without a row): vectors past its end read as zero, so the
      // values need no mask
      const __amdgpu_buffer_rsrc_t xrsrc = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<char*>(static_cast<const char*>(xv) + static_cast<int64_t>(srow) * K * (16 / E)), 0,
          active ? K * (16 / E) : 0, 0x00020000);
#pragma unroll
      for (int p = 0; p < VP; ++p) {
        const int v = gtid + G * kWave * p;
        xr[p] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                              xrsrc, static_cast<uint32_t>(v * 16), 0, 0));
      }
    }
    // gamma through a buffer resource of size 0 when it is NULL: the loads
    // then return zeros without touching memory, and no branch separates them
    // from the weight loads that follow (so a wait for x and gamma need not
    // wait for the weights too)
    const __amdgpu_buffer_rsrc_t grsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(gamma), 0, gamma != nullptr ? K * 4 : 0, 0x00020000);
#pragma unroll
    for (int p = 0; p < VP; ++p) {
      const int v = gtid + G * kWave * p;
      const int sv = (active && v < nvec) ? v : 0;
#pragma unroll
      for (int e4 = 0; e4 < E / 4; ++e4) {
        const uint32_t off = static_cast<uint32_t>((sv * E + 4 * e4) * 4);
        gr[p][e4] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(grsrc, off, 0, 0));
      }
    }
  }

  // values of vector p as fp32 (zero outside the row)
  __device__ __forceinline__ void values(int p, float* f) const {
    const int v = gtid + G * kWave * p;
    const bool ok = active && v < nvec;
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
        f[e] = ok ? mlgru_out_gate(gv[e], hn[e]) : 0.0f;
      }
      // the new state, once per call: workgroup 0 stores it
      if (ok && h_out != nullptr && blockIdx.x == 0)
        *reinterpret_cast<float4*>(h_out + static_cast<int64_t>(row) * (nvec * 4) + v * 4) =
            make_float4(hn[0], hn[1], hn[2], hn[3]);
    } else if constexpr (E == 8) {  // zero past the row's end (see load)
      const uint32_t w[4] = {xr[p].x, xr[p].y, xr[p].z, xr[p].w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f[2 * i] = __uint_as_float(w[i] << 16);
        f[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
      }
    } else {
      f[0] = __uint_as_float(xr[p].x);
      f[1] = __uint_as_float(xr[p].y);
      f[2] = __uint_as_float(xr[p].z);
      f[3] = __uint_as_float(xr[p].w);
    }
  }
  __device__ __forceinline__ float gamma_at(int p, int e) const {
    const float4 g = gr[p][e / 4];
    const int k = e % 4;
    return k == 0 ? g.x : k == 1 ? g.y : k == 2 ? g.z : g.w;
  }

  // RMSNorm, absmax and quantisation of the staged values into LDS, in two
  // parts.  begin(): the local sum of squares and its wave reduction (this is
  // where a row wave first waits for its activations).  finish(): two block
  // barriers, which every wave reaches, while only the waves of a row group
  // do the work (`active` is uniform across a wave).  The row sum of q is
  // left in the per-wave slots.
  float f[VP][E];
  __device__ __forceinline__ void begin(const Shared& sh) {
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

  __device__ __forceinline__ void finish(bool has_gamma, int K, const Shared& sh, bool first_barrier = true) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int w0 = row * G;
    if (first_barrier) __syncthreads();
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
    __syncthreads();
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
// past the end of q), a_scale and q_rowsum by the first MT threads.  The copy
// is complete once the issuing wave has waited for all its vector memory
// operations and passed a barrier.
constexpr int kBufferFlags = 0x00020000;  // gfx9 buffer descriptor word 3
typedef int v4i __attribute__((ext_vector_type(4)));

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

template <int MT>
struct QStage {
  float a;
  int rs;
  __device__ __forceinline__ void load(const int8_t* __restrict__ q, const float* __restrict__ a_scale,
                                       const int32_t* __restrict__ q_rowsum, int K, const Shared& sh) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int bytes = MT * K;
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
    const int t = threadIdx.x < MT ? threadIdx.x : 0;
    a = a_scale != nullptr ? a_scale[t] : 0.0f;
    rs = q_rowsum[t];
  }
  __device__ __forceinline__ void store(const Shared& sh) const {
    // every LDS-DMA write of this wave has landed
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0); no wait on the other counters
    const int t = threadIdx.x < MT ? threadIdx.x : 0;
    sh.a_scale[t] = a;
    sh.rowsum[t] = rs;
  }
};

// Weight loads go through a buffer resource (base and size in SGPRs): the
// load takes the lane's 32-bit offset in a VGPR and the slot's offset in an
// SGPR, so no vector address arithmetic is spent per slot, and the hardware
// range check returns 0 past the end of the packed array.

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
  int q_bytes;
  int q_stride;
  Affine affine;
  const float* h_in;  // kMlgru
  float* h_out;       // kMlgru
};

// The weights of a workgroup's columns are streamed in "slots": wave w owns
// the word rows [jb, je), both multiples of H (H divides K/16), and slot s of
// lane (c, h) is word row jb + H s + h.  Whether a slot exists is therefore
// the same for the whole wave, and its address is a scalar base
// (Wp + (jb + H s) N) plus a per-lane offset (h N + column) computed once.
//
// kLdsW: the workgroup's whole weight block (K/16 word rows of 64 columns) is
// copied into LDS by LDS-DMA at entry -- 16 bytes per lane, four word rows
// per wave instruction, no registers held, everything in flight at once --
// by the waves that do not normalise token rows (H = 1, at most 2 tokens),
// so the norm's own LDS traffic never waits on the copies; the contraction
// then reads the words from LDS.
template <int MT, int H, Src S, int VP, int kPrefetch, Epilogue EP, bool kLdsW = false, bool kMfma = false>
__global__ __launch_bounds__(kThreads) void decode_kernel(const Params prm) {
  static_assert(kMfma || kPrefetch % 4 == 0, "prefetch goes in groups of four");
  static_assert(!(kMfma && kLdsW), "the matrix-core contraction streams its words from memory");
  static_assert(!kLdsW || (H == 1 && MT <= 2 && S != Src::kQuantised), "LDS weight staging: H = 1, <= 2 tokens");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int K = prm.K;
  const int64_t N = prm.N;
  const Shared sh = carve(smem, prm.q_bytes, prm.q_stride);
  static_assert(S != Src::kMlgru || EP == Epilogue::kAffineF32, "the MLGRU prologue feeds the output projection");
  // read at entry: its latency then overlaps the rest of the kernel
  const float wscale = (EP == Epilogue::kDequantF32 || EP == Epilogue::kGluF32) ? prm.w_scale[0] : 0.0f;
  const float wscale_u = EP == Epilogue::kGluF32 ? prm.w_scale[1] : 0.0f;
  static_assert(EP != Epilogue::kAffineF32 || S != Src::kQuantised, "affine epilogue from x only");
  constexpr int C = kWave / H;  // columns per workgroup
  static_assert(EP != Epilogue::kGluF32 || (C >= 32 && S != Src::kQuantised && S != Src::kMlgru),
                "GLU output: whole gate/up block pairs per workgroup, activations from x");
  // kMfma: F = C / 16 column blocks of 16; a slot is one k64 step (4 word
  // rows), lane (g, l16) reading word row 4 s + g of columns F l16 .. + F - 1
  constexpr int F = C / 16;
  constexpr int RS = kMfma ? 4 : H;  // word rows per slot
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = lane % C, h = lane / C;
  const int l16 = lane & 15, g16 = lane >> 4;
  const int64_t n = kMfma ? static_cast<int64_t>(blockIdx.x) * C + F * l16
                          : static_cast<int64_t>(blockIdx.x) * C + c;
  const bool col_ok = n < N;
  const int J = K / 16;
  const int per_wave = ((J + kWaves * RS - 1) / (kWaves * RS)) * RS;
  const int jb = min(wave * per_wave, J);
  const int je = min(jb + per_wave, J);
  const int ns = kMfma ? (je - jb + 3) / 4 : (je - jb) / H;  // slots of this wave (uniform)
  // byte offsets from Wp: packed weights are < 4 GiB
  const __amdgpu_buffer_rsrc_t wrsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(prm.Wp), 0, static_cast<int>(static_cast<uint32_t>(J) * 4u * static_cast<uint32_t>(N)),
      kBufferFlags);
  const uint32_t row_bytes = 4u * static_cast<uint32_t>(N);
  const uint32_t lane_off = static_cast<uint32_t>(kMfma ? g16 : h) * row_bytes +
                            4u * static_cast<uint32_t>(col_ok ? n : 0);
  const uint32_t slot_bytes = static_cast<uint32_t>(RS) * row_bytes;
  const uint32_t wave_bytes = static_cast<uint32_t>(jb) * row_bytes;

  // 1. activation loads.  The waves that normalise the token rows wait for
  //    them and reduce sum x^2 before any weight load is issued, and every
  //    wave waits for that: x and gamma then cross a quiet memory system
  //    (issued together with 3 MB of weight misses they return late), and
  //    the rest of the norm overlaps the weight stream.
  if constexpr (kLdsW) {
    // word rows 4g .. 4g + 3 of the block: lane l copies row 4g + l / 16,
    // columns 4 (l % 16) .. + 3 (N % 4 == 0: a 16-byte chunk is whole); rows
    // past K/16 fall outside the buffer and read as zero; columns past N
    // belong to outputs that are not stored.
    // Issued first, by the waves that do no row work; those waves then issue
    // no other vector memory load before the wait ahead of the contraction,
    // so no wait the compiler places (it cannot see these copies) holds them
    // up at the norm's barriers.  The copies are inline assembly, out of the
    // compiler's sight:
    // it would otherwise hold every barrier of the norm until they land.
    // Loads retire in issue order, so the compiler's own waits can only wait
    // longer because of them, never shorter; the wait for the copies
    // themselves is the explicit vmcnt(0) before the contraction.
    if (wave >= row_waves<MT>() * row_groups<MT>()) {
      const int first = wave - row_waves<MT>() * row_groups<MT>();
      const int issuers = kWaves - row_waves<MT>() * row_groups<MT>();
      const int G = (J + 3) / 4;
      const uint32_t n0 = static_cast<uint32_t>(blockIdx.x) * kWave;
      const uint32_t lv = (static_cast<uint32_t>(lane >> 4) * static_cast<uint32_t>(N) + n0 +
                           4u * static_cast<uint32_t>(lane & 15)) * 4u;
      const uint64_t wa = reinterpret_cast<uint64_t>(prm.Wp);
      const v4i desc = {static_cast<int>(static_cast<uint32_t>(wa)), static_cast<int>((wa >> 32) & 0xFFFF),
                        static_cast<int>(static_cast<uint32_t>(J) * 4u * static_cast<uint32_t>(N)), kBufferFlags};
      const uint32_t wl = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(smem)) +
                          static_cast<uint32_t>(prm.q_bytes + kScalarBytes);
      for (int g = first; g < G; g += issuers) {  // wave-uniform
        const uint32_t dst = __builtin_amdgcn_readfirstlane(wl + static_cast<uint32_t>(g * kLdsDmaChunk));
        const uint32_t soff = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(g) * 4u * row_bytes);
        asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                     :
                     : "s"(dst), "v"(lv), "s"(desc), "s"(soff)
                     : "memory", "m0");
      }
    }
  }
  RowStage<MT, S == Src::kQuantised ? Src::kBf16 : S, VP> rows;
  QStage<MT> qs;
  if constexpr (S == Src::kQuantised) {
    qs.load(prm.q, prm.a_scale, prm.q_rowsum, K, sh);
  } else {
    rows.load(prm.x, prm.gamma, K, kLdsW, prm.h_in, prm.h_out);
  }
  // the factors of the column this thread writes in the affine epilogue
  // (issued after the token rows, so a wait for those leaves them in flight)
  ColAffine col{};
  if constexpr (EP == Epilogue::kAffineF32) {
    if (!kLdsW || tid < MT * C) {  // under kLdsW: the epilogue's threads only (row waves)
      const int64_t cn = static_cast<int64_t>(blockIdx.x) * C + tid % C;
      col = load_col_affine(prm.affine, prm.w_scale, static_cast<uint32_t>(N),
                            cn < N ? static_cast<uint32_t>(cn) : 0u);
    }
  }
  if constexpr (S != Src::kQuantised) {
    if constexpr (kWeightDelay < 0) {
      rows.begin(sh);
      __syncthreads();
    } else {
      rows.begin(sh);
      if (!rows.active) __builtin_amdgcn_s_sleep(kWeightDelay);
    }
  }
  __builtin_amdgcn_sched_barrier(0);

  // 2. every weight slot of the first prefetch group, straight-line code
  //    (loads retire in issue order, so later waits can count them).  Slots
  //    past the wave's range repeat its last slot (they are not used); a wave
  //    without slots reads past the end of the buffer, which returns zeros
  //    without a memory access.
  uint32_t wbuf[kPrefetch];
  Words<F> wmf[kPrefetch];
  const int last = ns > 0 ? ns - 1 : 0;
  if constexpr (kMfma) {
#pragma unroll
    for (int p = 0; p < kPrefetch; ++p) {
      const uint32_t sp = static_cast<uint32_t>(p < last ? p : last);
      wmf[p] = load_words<F>(wrsrc, lane_off, wave_bytes + sp * slot_bytes);
    }
  } else if constexpr (!kLdsW) {
#pragma unroll
    for (int p = 0; p < kPrefetch; ++p) {
      const uint32_t sp = static_cast<uint32_t>(p < last ? p : last);
      wbuf[p] = __builtin_amdgcn_raw_buffer_load_b32(wrsrc, lane_off, wave_bytes + sp * slot_bytes, 0);
    }
  }
  __builtin_amdgcn_sched_barrier(0);

  // 3. quantised activations into LDS (waits for the activation loads only)
  if constexpr (kLdsW) {
    constexpr int kRowThreads = row_waves<MT>() * row_groups<MT>() * kWave;
    if (tid < kRowThreads)
      for (int i = tid; i < kMaxTokens * kRedStride; i += kRowThreads) sh.red[i] = 0;
  } else {
    if (tid < kMaxTokens * kRedStride) sh.red[tid] = 0;
  }
  if constexpr (S == Src::kQuantised) {
    qs.store(sh);
  } else {
    rows.finish(prm.gamma != nullptr, K, sh, kWeightDelay >= 0);
  }
  // every LDS-DMA copy of this wave has landed before the barrier
  if constexpr (kLdsW) __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  __syncthreads();

  // 4. contraction.  A slot past the wave's range gets the word 0 (code 0
  // for every k, so its dot products add nothing) and reads q at a valid
  // row, which keeps the loop free of branches; the q vectors of the next
  // word are read from LDS while the current word is accumulated.
  int acc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[m] = 0;
  if constexpr (kLdsW) {
    const uint32_t* wl = reinterpret_cast<const uint32_t*>(smem + prm.q_bytes + kScalarBytes);
#pragma unroll 4
    for (int s = 0; s < ns; ++s) {
      const int j = jb + s;
      const uint32_t w = wl[j * kWave + c];
      const uint32_t c0 = codes4(w, 0), c1 = codes4(w, 1), c2 = codes4(w, 2), c3 = codes4(w, 3);
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        const uint4 q4 = *reinterpret_cast<const uint4*>(sh.q + m * K + 16 * j);
        int a = acc[m];
        a = dot4(c0, q4.x, a);
        a = dot4(c1, q4.y, a);
        a = dot4(c2, q4.z, a);
        a = dot4(c3, q4.w, a);
        acc[m] = a;
      }
    }
  }
  if constexpr (kMfma) {
    // 16 x 16 x 64 int8 matrix-core products: the code bytes of F column
    // blocks (first operand, rows = columns F i + f) against the token rows
    // of q (second operand, rows l16 < MT; the others and word rows past K/16
    // give zeros).  Lane (g, l16) ends with block f's columns F (4 g + r) + f,
    // r < 4, of token l16.
    v4i accf[F];
#pragma unroll
    for (int f = 0; f < F; ++f) accf[f] = v4i{0, 0, 0, 0};
    const bool tok = l16 < MT;
    const int8_t* qrow = sh.q + (tok ? l16 : 0) * sh.q_stride;
    for (int base = 0; base < ns; base += kPrefetch) {
      Words<F> cur[kPrefetch];
#pragma unroll
      for (int p = 0; p < kPrefetch; ++p) cur[p] = wmf[p];
      const int nb = base + kPrefetch;
      if (nb < ns) {
#pragma unroll
        for (int p = 0; p < kPrefetch; ++p) {
          const uint32_t sp = static_cast<uint32_t>(nb + p < ns ? nb + p : ns - 1);
          wmf[p] = load_words<F>(wrsrc, lane_off, wave_bytes + sp * slot_bytes);
        }
      }
#pragma unroll
      for (int p = 0; p < kPrefetch; ++p) {
        const int j = jb + 4 * (base + p) + g16;
        const bool ok = tok && base + p < ns && j < J;
        const uint4 qv = *reinterpret_cast<const uint4*>(qrow + 16 * (j < J ? j : J - 1));
        const v4i qf = ok ? __builtin_bit_cast(v4i, qv) : v4i{0, 0, 0, 0};
#pragma unroll
        for (int f = 0; f < F; ++f) {
          const uint32_t w = cur[p].w[f];
          const v4i cw = {static_cast<int>(codes4(w, 0)), static_cast<int>(codes4(w, 1)),
                          static_cast<int>(codes4(w, 2)), static_cast<int>(codes4(w, 3))};
          accf[f] = __builtin_amdgcn_mfma_i32_16x16x64_i8(cw, qf, accf[f], 0, 0, 0);
        }
      }
    }
    if (tok) {
#pragma unroll
      for (int f = 0; f < F; ++f)
#pragma unroll
        for (int r = 0; r < 4; ++r) atomicAdd(&sh.red[l16 * kRedStride + F * (4 * g16 + r) + f], accf[f][r]);
    }
  }
  for (int base = 0; base < ((kLdsW || kMfma) ? 0 : ns); base += kPrefetch) {
    uint32_t cur[kPrefetch];
#pragma unroll
    for (int p = 0; p < kPrefetch; ++p) cur[p] = base + p < ns ? wbuf[p] : 0u;
    const int nb = base + kPrefetch;
#pragma unroll
    for (int p0 = 0; p0 < kPrefetch; p0 += 4) {
      if (nb + p0 < ns) {
#pragma unroll
        for (int p = p0; p < p0 + 4; ++p) {
          const uint32_t sp = static_cast<uint32_t>(nb + p < ns ? nb + p : ns - 1);
          wbuf[p] = __builtin_amdgcn_raw_buffer_load_b32(wrsrc, lane_off, wave_bytes + sp * slot_bytes, 0);
        }
      }
    }
    auto q_at = [&](int p, int m) -> uint4 {
      const int j = base + p < ns ? jb + H * (base + p) + h : jb + h;
      return *reinterpret_cast<const uint4*>(sh.q + m * K + 16 * j);
    };
    uint4 qv[2][MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) qv[0][m] = q_at(0, m);
#pragma unroll
    for (int p = 0; p < kPrefetch; ++p) {
      if (p + 1 < kPrefetch) {
#pragma unroll
        for (int m = 0; m < MT; ++m) qv[(p + 1) & 1][m] = q_at(p + 1, m);
      }
      const uint32_t w = cur[p];
      const uint32_t c0 = codes4(w, 0), c1 = codes4(w, 1), c2 = codes4(w, 2), c3 = codes4(w, 3);
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        const uint4 q4 = qv[p & 1][m];
        int a = acc[m];
        a = dot4(c0, q4.x, a);
        a = dot4(c1, q4.y, a);
        a = dot4(c2, q4.z, a);
        a = dot4(c3, q4.w, a);
        acc[m] = a;
      }
    }
  }

  // 5. column sums over (wave, h) with LDS atomics, then dequantise
  if constexpr (!kMfma) {
#pragma unroll
    for (int m = 0; m < MT; ++m) atomicAdd(&sh.red[m * kRedStride + c], acc[m]);
  }
  __syncthreads();
  if constexpr (EP == Epilogue::kGluF32) {
    // The packed columns alternate 16 gate and 16 up columns, and a
    // workgroup's C columns are C / 32 whole pairs: thread (m, channel) forms
    // SiLU(g) * u of its channel (the formula and order of the MFMA kernel's
    // GLU epilogue, so both give the same bits) into the L = N / 2 wide output.
    constexpr int kHalf = C / 2;
    if (tid < MT * kHalf) {
      const int m = tid / kHalf, hc = tid % kHalf;
      const int cg = (hc / 16) * 32 + hc % 16;  // gate column; up column cg + 16
      const int64_t L = N / 2;
      const int64_t ch = static_cast<int64_t>(blockIdx.x) * kHalf + hc;
      constexpr int G = row_waves<MT>();
      int rsum = 0;
#pragma unroll
      for (int w = 0; w < G; ++w) rsum += sh.slot_i[m * G + w];
      if (ch < L) {
        const float sg = sh.a_scale[m] * wscale, su = sh.a_scale[m] * wscale_u;
        const float gv = static_cast<float>(sh.red[m * kRedStride + cg] - rsum) * sg;
        const float uv = static_cast<float>(sh.red[m * kRedStride + cg + 16] - rsum) * su;
        static_cast<float*>(prm.out)[m * L + ch] = gv * sigmoid_hw(gv) * uv;
      }
    }
  } else if (tid < MT * C) {
    const int m = tid / C, cc = tid % C;
    const int64_t nn = static_cast<int64_t>(blockIdx.x) * C + cc;
    int rsum;
    if constexpr (S == Src::kQuantised) {
      rsum = sh.rowsum[m];
    } else {
      constexpr int G = row_waves<MT>();
      rsum = 0;
#pragma unroll
      for (int w = 0; w < G; ++w) rsum += sh.slot_i[m * G + w];
    }
    if (nn < N) {
      const int v = sh.red[m * kRedStride + cc] - rsum;
      if constexpr (EP == Epilogue::kDequantF32) {
        static_cast<float*>(prm.out)[m * N + nn] = static_cast<float>(v) * (sh.a_scale[m] * wscale);
      } else if constexpr (EP == Epilogue::kAffineF32) {
        const float z = static_cast<float>(v) * (sh.a_scale[m] * col.ws) + col.bias;
        static_cast<float*>(prm.out)[m * N + nn] = affine_act(z, col.act, col.lb);
      } else
        static_cast<int32_t*>(prm.out)[m * N + nn] = v;
    }
  }
}

// q row stride in LDS.  The matrix-core contraction reads 16 bytes of one k
// group from each token row at once; rows padded by 16 bytes put those reads
// on distinct banks.  Pre-quantised q is copied in whole 1 KB chunks, so it
// is padded only when a chunk never straddles two rows (K % 1024 == 0).
inline int q_stride_for(bool mfma, bool quantised, int K) {
  return (mfma && (!quantised || K % kLdsDmaChunk == 0)) ? K + 16 : K;
}

template <int MT, int H, Src S, int VP, int PF, Epilogue EP, bool kLdsW = false, bool kMfma = false>
hipError_t launch_one(const DecodeArgs& a, hipStream_t stream) {
  constexpr int C = kWave / H;
  // the q region is whole LDS-DMA chunks
  const int q_stride = q_stride_for(kMfma, S == Src::kQuantised, a.K);
  const int region = ((MT * q_stride + kLdsDmaChunk - 1) / kLdsDmaChunk) * kLdsDmaChunk;
  const dim3 grid(static_cast<unsigned>((a.N + C - 1) / C));
  const Params prm{a.Wpacked, a.x, a.gamma, a.q, a.a_scale, a.q_rowsum, a.w_scale, a.out,
                   a.N, a.K, region, q_stride, a.affine, a.h_in, a.h_out};
  const int wbytes = kLdsW ? ((a.K / 16 + 3) / 4) * kLdsDmaChunk : 0;
  hipLaunchKernelGGL((decode_kernel<MT, H, S, VP, PF, EP, kLdsW, kMfma>), grid, dim3(kThreads),
                     region + kScalarBytes + wbytes, stream, prm);
  return hipGetLastError();
}

// Weight words in flight per lane: a wave's whole range when it holds at most
// four slots, else eight at a time (measured: deeper prefetch only delays
// the loads of the waves that also normalise the token rows).  Matrix-core
// contraction: slots are k64 steps of F words each, two or four in flight.
template <int MT, int H, Src S, int VP, Epilogue EP, bool kMfma>
hipError_t dispatch_pf(const DecodeArgs& a, hipStream_t stream) {
  const int J = a.K / 16;
  if constexpr (kMfma) {
    const int steps = (J + kWaves * 4 - 1) / (kWaves * 4);
    if (steps <= 2) return launch_one<MT, H, S, VP, 2, EP, false, true>(a, stream);
    return launch_one<MT, H, S, VP, 4, EP, false, true>(a, stream);
  } else {
    const int slots = (J + kWaves * H - 1) / (kWaves * H);
    if (slots <= 4) return launch_one<MT, H, S, VP, 4, EP>(a, stream);
    return launch_one<MT, H, S, VP, 8, EP>(a, stream);
  }
}

// vectors of 16 bytes per thread a row needs: ceil(K / E / (G * 64))
inline int needed_vp(int64_t mt, int K, bool f32) {
  const int64_t p = mt <= 1 ? 1 : mt <= 2 ? 2 : mt <= 4 ? 4 : 8;
  const int64_t g = kWaves / p < kMaxRowWaves ? kWaves / p : kMaxRowWaves;
  const int64_t lanes = g * kWave;
  const int64_t nvec = K / (f32 ? 4 : 8);
  return static_cast<int>((nvec + lanes - 1) / lanes);
}

template <int MT, int H, Src S, Epilogue EP, bool kMfma = false>
hipError_t dispatch_vp(const DecodeArgs& a, hipStream_t stream) {
  if constexpr (S == Src::kQuantised) {
    return dispatch_pf<MT, H, S, 1, EP, kMfma>(a, stream);
  } else {
    const int vp = needed_vp(MT, a.K, S == Src::kF32 || S == Src::kMlgru);
    if (vp <= 1) return dispatch_pf<MT, H, S, 1, EP, kMfma>(a, stream);
    if (vp <= 2) return dispatch_pf<MT, H, S, 2, EP, kMfma>(a, stream);
    if (vp <= 4) return dispatch_pf<MT, H, S, 4, EP, kMfma>(a, stream);
    return hipErrorInvalidValue;  // excluded by decode_fits
  }
}

// The LDS weight staging pays when a workgroup's block is large (many word
// rows per lane); it needs N % 4 == 0 (16-byte row chunks) and room in LDS
// next to the q region.
constexpr int kLdsWMinRows = 256;
constexpr int kLdsLimit = 160 * 1024;
inline bool use_lds_weights(int mt, int K, int64_t N, bool from_x) {
  const int J = K / 16;
  if (!from_x || mt > 2 || N % 4 != 0 || J < kLdsWMinRows) return false;
  const int region = ((mt * K + kLdsDmaChunk - 1) / kLdsDmaChunk) * kLdsDmaChunk;
  return region + kScalarBytes + ((J + 3) / 4) * kLdsDmaChunk <= kLdsLimit;
}

template <int MT, Src S, Epilogue EP>
hipError_t dispatch_h(const DecodeArgs& a, hipStream_t stream) {
  if constexpr (MT <= 2 && S != Src::kQuantised) {
    if (use_lds_weights(MT, a.K, a.N, true)) {
      const int vp = needed_vp(MT, a.K, S == Src::kF32 || S == Src::kMlgru);
      if (vp <= 1) return launch_one<MT, 1, S, 1, 4, EP, true>(a, stream);
      if (vp <= 2) return launch_one<MT, 1, S, 2, 4, EP, true>(a, stream);
      if (vp <= 4) return launch_one<MT, 1, S, 4, 4, EP, true>(a, stream);
    }
  }
  // Two or more tokens: the matrix cores.  Each packed word (16 weights)
  // costs 4 MT v_dot4 on the vector ALU, and at 8 tokens that work alone
  // takes longer than streaming the weights; one 16x16x64 MFMA covers four
  // words of 16 columns for 16 token rows.  Column blocks per workgroup: as few as
  // keep the grid within one round of the CUs, with loads aligned to their
  // width (N % F == 0).
  constexpr bool kGlu = EP == Epilogue::kGluF32;  // needs C >= 32 (N % 32 == 0)
  if constexpr (MT >= kMfmaMinTokens) {
    const int64_t N = a.N;
    if constexpr (!kGlu) {
      if ((N + 15) / 16 <= kGridRound) return dispatch_vp<MT, 4, S, EP, true>(a, stream);
    }
    if (N % 2 == 0 && ((N + 31) / 32 <= kGridRound || N % 4 != 0))
      return dispatch_vp<MT, 2, S, EP, true>(a, stream);
    if (N % 4 == 0) return dispatch_vp<MT, 1, S, EP, true>(a, stream);
    if constexpr (!kGlu) return dispatch_vp<MT, 4, S, EP, true>(a, stream);
    return hipErrorInvalidValue;
  }
  // A 1024-thread workgroup fills a CU, so the grid should stay within one
  // round of the 256 CUs: the most lanes per column (more workgroups, fewer
  // words per lane) that still does and that divides K/16.
  const int J = a.K / 16;
  if constexpr (!kGlu) {
    if (J % 4 == 0 && (a.N + 15) / 16 <= kGridRound) return dispatch_vp<MT, 4, S, EP>(a, stream);
  }
  if (J % 2 == 0 && (a.N + 31) / 32 <= kGridRound) return dispatch_vp<MT, 2, S, EP>(a, stream);
  return dispatch_vp<MT, 1, S, EP>(a, stream);
}

template <Src S, Epilogue EP>
hipError_t dispatch_mt(int mt, const DecodeArgs& a, hipStream_t stream) {
  switch (mt) {
    case 1: return dispatch_h<1, S, EP>(a, stream);
    case 2: return dispatch_h<2, S, EP>(a, stream);
    case 3: return dispatch_h<3, S, EP>(a, stream);
    case 4: return dispatch_h<4, S, EP>(a, stream);
    case 5: return dispatch_h<5, S, EP>(a, stream);
    case 6: return dispatch_h<6, S, EP>(a, stream);
    case 7: return dispatch_h<7, S, EP>(a, stream);
    case 8: return dispatch_h<8, S, EP>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

bool decode_fits(int64_t mt, int K, int64_t N, bool from_x, bool x_is_f32) {
  if (mt < 1 || mt > kMaxTokens || mt * K > kDecodeMaxLdsQ) return false;
  // 32-bit offsets: the packed array plus the slack of clamped slot offsets
  if (static_cast<int64_t>(K / 16 + 8) * N * 4 >= (int64_t(1) << 32)) return false;
  if (!from_x) return true;
  return needed_vp(mt, K, x_is_f32) <= 4;
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream) {
  const int mt = static_cast<int>(a.M);  // 1..8; the caller slices larger M
  if (a.epilogue == Epilogue::kGluF32) {
    if (a.q != nullptr || a.mlgru_in || a.N % 32 != 0) return hipErrorInvalidValue;
    if (a.x_is_f32) return dispatch_mt<Src::kF32, Epilogue::kGluF32>(mt, a, stream);
    return dispatch_mt<Src::kBf16, Epilogue::kGluF32>(mt, a, stream);
  }
  if (a.epilogue == Epilogue::kAffineF32) {
    if (a.q != nullptr) return hipErrorInvalidValue;
    if (a.mlgru_in) return dispatch_mt<Src::kMlgru, Epilogue::kAffineF32>(mt, a, stream);
    if (a.x_is_f32) return dispatch_mt<Src::kF32, Epilogue::kAffineF32>(mt, a, stream);
    return dispatch_mt<Src::kBf16, Epilogue::kAffineF32>(mt, a, stream);
  }
  if (a.q != nullptr) {
    if (a.epilogue == Epilogue::kDequantF32)
      return dispatch_mt<Src::kQuantised, Epilogue::kDequantF32>(mt, a, stream);
    return dispatch_mt<Src::kQuantised, Epilogue::kRawI32>(mt, a, stream);
  }
  if (a.x_is_f32) return dispatch_mt<Src::kF32, Epilogue::kDequantF32>(mt, a, stream);
  return dispatch_mt<Src::kBf16, Epilogue::kDequantF32>(mt, a, stream);
}

}  // namespace mmf
