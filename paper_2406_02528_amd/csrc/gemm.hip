// Prefill contraction (any M, built for M in the thousands): the ternary sum
// as a dense int8 contraction on the gfx950 matrix cores.
//
// At thousands of tokens the ternary accumulation is a dense contraction of
// int8 activations against {-1,0,1} weights, so it runs on
// v_mfma_i32_32x32x32_i8 with exact int32 accumulation.  The weight operand is
// the code c = t + 1 in {0,1,2}; the epilogue subtracts sum_k q (sum q*t =
// sum q*c - sum q) and dequantises.
//
// Operands and pipeline:
//  - Each workgroup computes a BM x BN output tile.  Its operands stream
//    through an S-slot LDS ring, one slot per BK-deep k stage: A (q, int8
//    [M][K]) as BM rows of BK bytes, B as BK/16 rows of BN packed words.
//  - The global->LDS copies are LDS-DMA buffer loads (the data goes straight
//    from the memory pipeline into LDS without passing through registers), so
//    S - 1 stages are in flight while the matrix cores work on the oldest.
//  - B stays packed until it reaches the registers: for a 32x32x32 MFMA,
//    lane l supplies column l % 32 and the 16 k-values of group l / 32, which
//    is exactly one packed word Wpacked[j][n], expanded in registers into four
//    dwords of code bytes right before use.
//  - Both operands are read through buffer resources, whose range check
//    returns zero past the end of the array (rows past M, chunks past K, word
//    rows past K/16) without touching memory.
//  - Fragment reads of the next k32 step are interleaved with the MFMAs of
//    the current one (double-buffered fragment registers).
//
// Tile order: workgroups are dealt round-robin to the 8 XCDs, each with its
// own L2, so the linear workgroup id is remapped to give every XCD a
// contiguous run of tiles, walked in groups of kGroupM tile rows; the tiles
// an XCD works on at once then share A rows and B columns in its L2.
#include "mmf_device.h"
#include "mmf_launch.h"

namespace mmf {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kBufferFlags = 0x00020000;  // gfx9 buffer descriptor word 3
constexpr int kXcds = 8;
constexpr int kGroupM = 4;

__device__ __forceinline__ void tile_coords(int64_t tiles_m, int64_t tiles_n, int64_t& tm,
                                            int64_t& tn) {
  const int64_t total = tiles_m * tiles_n;
  const int64_t b = blockIdx.x;
  // XCD-contiguous logical index: XCD x (= b % 8) takes tiles
  // [x * per, (x + 1) * per); the tail beyond 8 * per keeps its order.
  const int64_t per = total / kXcds;
  int64_t L = b;
  if (b < per * kXcds) L = (b % kXcds) * per + b / kXcds;
  // grouped row-major walk: kGroupM tile rows at a time, columns inside
  const int64_t group = L / (kGroupM * tiles_n);
  const int64_t first_m = group * kGroupM;
  const int64_t gm = (tiles_m - first_m) < kGroupM ? (tiles_m - first_m) : kGroupM;
  const int64_t in_group = L - group * kGroupM * tiles_n;
  tm = first_m + in_group % gm;
  tn = in_group / gm;
}

// s_waitcnt immediates (gfx9 encoding): at most n vector memory operations
// outstanding; with LGKM0 also every LDS operation completed, without it no
// wait on LDS (lgkmcnt field at its maximum).
#define MMF_WAIT_VM(n) (((n) & 0xF) | (0x7 << 4) | (0xF << 8) | ((((n) >> 4) & 3) << 14))
#define MMF_WAIT_VM_LGKM0(n) (((n) & 0xF) | (0x7 << 4) | ((((n) >> 4) & 3) << 14))

template <int BM, int BN, int WM, int WN, int BK, int S>
struct Tiling {
  static constexpr int kWavesM = BM / WM, kWavesN = BN / WN;
  static constexpr int kWaves = kWavesM * kWavesN;
  static constexpr int kThreads = kWaves * kWave;
  static constexpr int FM = WM / 32, FN = WN / 32;   // MFMA tiles per wave
  static constexpr int KS = BK / 32;                 // k32 steps per stage
  static constexpr int kChunks = BK / 16;            // 16-byte chunks per A row
  // A stage: BM rows of BK bytes, unpadded (each LDS-DMA instruction writes
  // 1 KB contiguously), chunks XOR-swizzled per row against bank conflicts.
  static constexpr int kABytes = BM * BK;
  static constexpr int kAInstr = kABytes / 1024;     // 16-byte-per-lane loads
  // B stage: BK/16 word rows of BN words, each padded by 32 words.
  static constexpr int kBRow = BN + 32;              // words
  static constexpr int kBBytes = (BK / 16) * kBRow * 4;
  static constexpr int kBInstr = (BK / 16) * BN / 64; // 4-byte-per-lane loads
  static constexpr int kAPerWave = kAInstr / kWaves, kBPerWave = kBInstr / kWaves;
  static constexpr int kLoadsPerStage = kAPerWave + kBPerWave;
  static constexpr int kStageBytes = kABytes + kBBytes;
  static_assert(kAInstr % kWaves == 0 && kBInstr % kWaves == 0, "loads must split evenly");
  static_assert(S >= 3, "need at least three stages");
};

// Chunk swizzle of A rows: row r stores logical chunk c in slot c ^ swz(r).
// For BK = 64 (4 chunks per row) it keeps ds_read_b128 of 32 consecutive rows
// at one chunk conflict-free both when 8 lanes share 32 banks and when 16
// lanes share 64 banks.
template <int kChunks>
__device__ __forceinline__ int a_swz(int r) {
  return ((r >> 1) ^ (r >> 3)) & (kChunks - 1);
}

template <int BM, int BN, int WM, int WN, int BK, int S, Epilogue EP>
__global__ __launch_bounds__((Tiling<BM, BN, WM, WN, BK, S>::kThreads)) void gemm_kernel(
    const int8_t* __restrict__ q, const float* __restrict__ a_scale,
    const int32_t* __restrict__ q_rowsum, const uint32_t* __restrict__ Wp,
    const float* __restrict__ w_scale, void* __restrict__ out, int M, int K, int N) {
  using T = Tiling<BM, BN, WM, WN, BK, S>;
  constexpr int FM = T::FM, FN = T::FN, KS = T::KS;
  // S ring slots, then the tile's per-row dequantisation factors
  __shared__ __attribute__((aligned(16))) char smem[S * T::kStageBytes + 8 * BM];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / T::kWavesN, wn = wave % T::kWavesN;
  const int l32 = lane & 31;
  const int g = lane >> 5;  // k group of this lane inside one MFMA
  int64_t tm, tn;
  tile_coords((M + BM - 1) / BM, (N + BN - 1) / BN, tm, tn);
  const int m0 = static_cast<int>(tm) * BM;
  const int n0 = static_cast<int>(tn) * BN;
  const int J = K / 16;
  const int KT = (K + BK - 1) / BK;


  // Per-lane source offsets of this wave's LDS-DMA loads (k0 added per stage).
  // A instruction i: rows 16 (wave * kAPerWave + i) + lane / 4 ... for BK = 64
  // (BK / 16 chunks per row in general); the lane's LDS slot s holds the
  // row's logical chunk s ^ swz(row).
  constexpr int kRowsPerInstr = 1024 / BK;
  uint32_t a_src[T::kAPerWave];
  int a_chunk[T::kAPerWave];
#pragma unroll
  for (int i = 0; i < T::kAPerWave; ++i) {
    const int r = (wave * T::kAPerWave + i) * kRowsPerInstr + lane / T::kChunks;
    const int c = (lane % T::kChunks) ^ a_swz<T::kChunks>(r);
    a_chunk[i] = c * 16;
    a_src[i] = static_cast<uint32_t>(m0 + r) * static_cast<uint32_t>(K) + static_cast<uint32_t>(c * 16);
  }
  // B instruction i: word row jj = idx / (BN / 64), words q64 * 64 + lane
  uint32_t b_src[T::kBPerWave];
  int b_jj[T::kBPerWave], b_dst[T::kBPerWave];
#pragma unroll
  for (int i = 0; i < T::kBPerWave; ++i) {
    const int idx = wave * T::kBPerWave + i;
    const int jj = idx / (BN / 64), q64 = idx % (BN / 64);
    b_jj[i] = jj;
    b_dst[i] = jj * T::kBRow * 4 + q64 * 256;
    // columns past N read the next word row or zero; their outputs are dropped
    b_src[i] = 4u * (static_cast<uint32_t>(jj) * static_cast<uint32_t>(N) +
                     static_cast<uint32_t>(n0 + q64 * 64 + lane));
  }
  const uint32_t b_row = 4u * static_cast<uint32_t>(N);

  // Buffer descriptors for the LDS-DMA loads (gfx9 layout: 48-bit base,
  // stride 0, size in bytes, format word).
  const uint64_t qa = reinterpret_cast<uint64_t>(q), wa = reinterpret_cast<uint64_t>(Wp);
  const v4i adesc = {static_cast<int>(static_cast<uint32_t>(qa)), static_cast<int>((qa >> 32) & 0xFFFF),
                     static_cast<int>(static_cast<uint32_t>(M) * static_cast<uint32_t>(K)), kBufferFlags};
  const v4i bdesc = {static_cast<int>(static_cast<uint32_t>(wa)), static_cast<int>((wa >> 32) & 0xFFFF),
                     static_cast<int>(static_cast<uint32_t>(J) * static_cast<uint32_t>(N) * 4u), kBufferFlags};
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(smem));

  // Issue the loads of stage kt into ring slot kt % S.  The LDS-DMA loads are
  // written as inline assembly, so the compiler does not see LDS writes that
  // could alias its fragment reads (it would wait for every load in flight
  // before each read); this kernel orders them itself with explicit vmcnt
  // waits before its barriers.  Offsets at or past the end of a buffer (rows
  // past M, chunks past K, word rows past K/16, stages past the last) read
  // zero without touching memory.
  auto issue = [&](int kt) {
    const uint32_t base = lds0 + static_cast<uint32_t>((kt % S) * T::kStageBytes);
    const int k0 = kt * BK;
#pragma unroll
    for (int i = 0; i < T::kAPerWave; ++i) {
      const uint32_t off = (k0 + a_chunk[i] < K) ? a_src[i] + static_cast<uint32_t>(k0) : 0x80000000u;
      const uint32_t dst = __builtin_amdgcn_readfirstlane(base + (wave * T::kAPerWave + i) * 1024);
      asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                   :
                   : "s"(dst), "v"(off), "s"(adesc)
                   : "memory", "m0");
    }
    const int j0 = k0 / 16;
#pragma unroll
    for (int i = 0; i < T::kBPerWave; ++i) {
      const uint32_t off = (j0 + b_jj[i] < J) ? b_src[i] + static_cast<uint32_t>(j0) * b_row : 0x80000000u;
      const uint32_t dst = __builtin_amdgcn_readfirstlane(base + T::kABytes + b_dst[i]);
      asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, 0 offen lds"
                   :
                   : "s"(dst), "v"(off), "s"(bdesc)
                   : "memory", "m0");
    }
  };

  v16i acc[FM][FN];
#pragma unroll
  for (int a = 0; a < FM; ++a)
#pragma unroll
    for (int b = 0; b < FN; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0;

  // Fragments of one k32 step, double buffered across steps and across stage
  // boundaries: A operands straight from LDS, B as raw packed words (bw) and
  // as expanded code dwords (bf).
  v4i af[2][FM], bf[2][FN];
  uint32_t bw[2][FN];
  auto read_frags = [&](int kt, int ks, int slot) {
    const char* st = smem + (kt % S) * T::kStageBytes;
    const uint32_t* Bs = reinterpret_cast<const uint32_t*>(st + T::kABytes);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const int row = wm * WM + fm * 32 + l32;
      const int c = (ks * 2 + g) ^ a_swz<T::kChunks>(row);
      af[slot][fm] = *reinterpret_cast<const v4i*>(st + row * BK + c * 16);
    }
#pragma unroll
    for (int f = 0; f < FN; ++f) bw[slot][f] = Bs[(2 * ks + g) * T::kBRow + wn * WN + f * 32 + l32];
  };
  auto unpack = [&](int slot) {
#pragma unroll
    for (int f = 0; f < FN; ++f) {
      const uint32_t x = bw[slot][f];
      bf[slot][f] = v4i{static_cast<int>(codes4(x, 0)), static_cast<int>(codes4(x, 1)),
                        static_cast<int>(codes4(x, 2)), static_cast<int>(codes4(x, 3))};
    }
  };

  // Software pipeline.  Ring slot kt % S holds stage kt.  Stage kt + S - 1
  // is issued during stage kt, into the slot of stage kt - 1, at the stage's
  // transition point: in its last k32 step, after this wave's loads of stage
  // kt + 1 have landed (the S - 3 younger stages may stay in flight) and a
  // barrier has made every wave's stage-kt+1 data visible.  Every read of
  // slot kt - 1 has been consumed by an earlier MFMA or unpack, so it is
  // complete before the barrier and the slot can be refilled.
  //
  // Each k32 step is fenced into three phases the compiler may not reorder:
  // the LDS reads of the next step, the MFMAs of the first A fragment (which
  // cover the read latency), and the remaining MFMAs with the expansion of
  // the next step's B words slotted between them.
  constexpr int kFirst = FN;                     // MFMAs in phase 2
  constexpr int kRest = FM * FN - kFirst;        // MFMAs in phase 3
  constexpr int kUnpackValu = 7 * FN;            // VALU of one unpack
  // The tile's per-row dequantisation inputs (q_rowsum, then a_scale) go
  // into LDS by LDS-DMA too, one 64-row chunk per wave, ahead of the ring's
  // first stages, so the prologue's wait covers them and the epilogue finds
  // them there.  Rows past M read zero.
  {
    static_assert(2 * BM == 64 * T::kWaves, "one row-factor chunk per wave");
    const int arr = wave / (BM / 64), chunk = wave % (BM / 64);
    const int row = m0 + chunk * 64 + lane;
    const uint32_t off = row < M ? 4u * static_cast<uint32_t>(row) : 0x80000000u;
    const uint64_t base = arr == 0 ? reinterpret_cast<uint64_t>(q_rowsum) : reinterpret_cast<uint64_t>(a_scale);
    const int bytes = (arr == 0 || EP == Epilogue::kDequantF32) ? M * 4 : 0;
    const v4i desc = {static_cast<int>(static_cast<uint32_t>(base)), static_cast<int>((base >> 32) & 0xFFFF),
                      bytes, kBufferFlags};
    const uint32_t dst = __builtin_amdgcn_readfirstlane(
        lds0 + static_cast<uint32_t>(S * T::kStageBytes + arr * BM * 4 + chunk * 256));
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, 0 offen lds"
                 :
                 : "s"(dst), "v"(off), "s"(desc)
                 : "memory", "m0");
  }
#pragma unroll
  for (int p = 0; p < S - 1; ++p) issue(p);
  __builtin_amdgcn_s_waitcnt(MMF_WAIT_VM((S - 2) * T::kLoadsPerStage));
  __builtin_amdgcn_s_barrier();
  read_frags(0, 0, 0);
  unpack(0);
  int fb = 0;  // fragment buffer of the current step
  for (int kt = 0; kt < KT; ++kt) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      __builtin_amdgcn_sched_barrier(0);
      if (ks + 1 < KS) {
        read_frags(kt, ks + 1, fb ^ 1);
      } else {
        __builtin_amdgcn_s_waitcnt(MMF_WAIT_VM((S - 3) * T::kLoadsPerStage));
        __builtin_amdgcn_s_barrier();
        issue(kt + S - 1);
        // unconditional (after the last stage it reads a slot of zeros), so
        // that the loop body stays one block the fences can order
        read_frags(kt + 1, 0, fb ^ 1);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int f = 0; f < FN; ++f)
        acc[0][f] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[fb][0], bf[fb][f], acc[0][f], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int fm = 1; fm < FM; ++fm)
#pragma unroll
        for (int f = 0; f < FN; ++f)
          acc[fm][f] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[fb][fm], bf[fb][f], acc[fm][f], 0, 0, 0);
      unpack(fb ^ 1);
      if constexpr (kRest > 0) {
#pragma unroll
        for (int i = 0; i < kRest; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                                  // MFMA
          __builtin_amdgcn_sched_group_barrier(0x002, (kUnpackValu + kRest - 1) / kRest, 0);  // VALU
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      (void)kFirst;
      fb ^= 1;
    }
  }
  // no LDS-DMA write may still be in flight when the workgroup's LDS is freed
  __builtin_amdgcn_s_waitcnt(MMF_WAIT_VM_LGKM0(0));

  // ---- epilogue: lane holds column l32, rows 8*(r/4) + 4*g + r%4 ----
  const int* s_rsum = reinterpret_cast<const int*>(smem + S * T::kStageBytes);
  const float* s_scale = reinterpret_cast<const float*>(smem + S * T::kStageBytes + 4 * BM);
  const float ws = (EP == Epilogue::kDequantF32) ? w_scale[0] : 0.0f;
  __syncthreads();
  // Range-checked buffer stores: rows past M fall outside the output's
  // range, columns past N are sent there explicitly; no branches.
  const uint32_t out_bytes = static_cast<uint32_t>(M) * static_cast<uint32_t>(N) * 4u;
  const __amdgpu_buffer_rsrc_t orsrc =
      __builtin_amdgcn_make_buffer_rsrc(out, 0, static_cast<int>(out_bytes), kBufferFlags);
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int lr = wm * WM + fm * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
      const int rs = s_rsum[lr];
      const float sc = s_scale[lr] * ws;
      const uint32_t row_bytes = static_cast<uint32_t>(m0 + lr) * static_cast<uint32_t>(N) * 4u;
#pragma unroll
      for (int f = 0; f < FN; ++f) {
        const int n = n0 + wn * WN + f * 32 + l32;
        const uint32_t off = (m0 + lr < M && n < N) ? row_bytes + 4u * static_cast<uint32_t>(n) : 0x80000000u;
        const int v = acc[fm][f][r] - rs;
        if constexpr (EP == Epilogue::kDequantF32)
          __builtin_amdgcn_raw_buffer_store_b32(static_cast<uint32_t>(__float_as_int(static_cast<float>(v) * sc)),
                                                orsrc, off, 0, 0);
        else
          __builtin_amdgcn_raw_buffer_store_b32(static_cast<uint32_t>(v), orsrc, off, 0, 0);
      }
    }
  }
}

template <int BM, int BN, int WM, int WN, int BK, int S>
hipError_t launch_cfg(const ContractArgs& a, int64_t m_begin, int64_t m_rows, hipStream_t stream) {
  using T = Tiling<BM, BN, WM, WN, BK, S>;
  const int lds = 0;  // the ring is static LDS
  const int64_t gm = (m_rows + BM - 1) / BM;
  const int64_t gn = (a.N + BN - 1) / BN;
  const dim3 grid(static_cast<unsigned>(gm * gn));
  const dim3 block(T::kThreads);
  const int8_t* q = a.q + m_begin * a.K;
  const float* as = a.a_scale ? a.a_scale + m_begin : nullptr;
  const int32_t* rs = a.q_rowsum + m_begin;
  if (a.epilogue == Epilogue::kDequantF32)
    hipLaunchKernelGGL((gemm_kernel<BM, BN, WM, WN, BK, S, Epilogue::kDequantF32>), grid, block, lds, stream,
                       q, as, rs, a.Wpacked, a.w_scale,
                       static_cast<void*>(static_cast<float*>(a.out) + m_begin * a.N),
                       static_cast<int>(m_rows), a.K, static_cast<int>(a.N));
  else
    hipLaunchKernelGGL((gemm_kernel<BM, BN, WM, WN, BK, S, Epilogue::kRawI32>), grid, block, lds, stream,
                       q, as, rs, a.Wpacked, a.w_scale,
                       static_cast<void*>(static_cast<int32_t*>(a.out) + m_begin * a.N),
                       static_cast<int>(m_rows), a.K, static_cast<int>(a.N));
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(const ContractArgs& a, hipStream_t stream) {
  // 32-bit buffer offsets: a launch covers at most 2^31 - 1 bytes of q, of
  // packed weights and of output; taller problems run in row slices.
  const int64_t packed = static_cast<int64_t>(a.K / 16) * a.N * 4;
  if (packed >= (int64_t(1) << 31) || a.N > (int64_t(1) << 24)) return hipErrorInvalidValue;
  const int64_t by_q = ((int64_t(1) << 31) - 1) / a.K;
  const int64_t by_y = ((int64_t(1) << 31) - 1) / (4 * a.N);
  int64_t slice = by_q < by_y ? by_q : by_y;
  slice = (slice / 256) * 256;
  if (slice < 256) return hipErrorInvalidValue;
  for (int64_t m0 = 0; m0 < a.M; m0 += slice) {
    const int64_t rows = a.M - m0 < slice ? a.M - m0 : slice;
    const hipError_t e = launch_cfg<256, 256, 64, 128, 64, 4>(a, m0, rows, stream);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace mmf
