// Prefill contraction (any M, built for M in the thousands): the ternary sum
// as a dense int8 contraction on the gfx950 matrix cores.
//
// At thousands of tokens the ternary accumulation is a dense contraction of
// int8 activations against {-1,0,1} weights, so it runs on
// v_mfma_i32_16x16x64_i8 with exact int32 accumulation.  The weight operand is
// the code c = t + 1 in {0,1,2}; the epilogue subtracts sum_k q (sum q*t =
// sum q*c - sum q) and dequantises.
//
// Tiling: a workgroup of 8 waves computes a 128 x 512 output tile (256 x 256
// when N % 4 != 0); wave (wm, wn) owns a 128 x 64 block as 8 x 4 MFMA tiles
// of 16 x 16.  Each expanded weight fragment therefore feeds eight MFMAs,
// which keeps the VALU work of the 2-bit expansion small against the matrix
// work.  The wide tile moves fewer operand bytes per MAC into LDS than a
// square one (the int8 rows of q are the heavy operand, the 2-bit weight
// columns the light one): 32 KB per 128-deep stage for 128 x 512 against
// 40 KB for 256 x 256, and the global->LDS copies are what limits the loop.
// A problem with few such tiles (a short M, a narrow N) runs on 64 x 512 or
// 64 x 256 tiles instead (waves of 64 x 64 or 32 x 64), whichever finishes
// first by the rule of gemm_tile_choice: a lone tile's k loop is latency-
// bound, so more, smaller tiles on more CUs beat a few wide ones.
// Where the wide tile is chosen, K <= 4096, the epilogue is not the affine
// one and the wide tiles fill more than one round of the CUs (or most of one
// at K <= 2048: gemm_paired), the same area is covered by two 128 x 256
// workgroups of 4 waves per CU instead (75 KB of LDS each, the same 128 x 64
// per wave): a tile's output stores, which otherwise run after its k loop
// with the matrix cores idle, then overlap the other workgroup's k loop.  The
// narrower tile moves 1.5x the operand bytes per MAC, a cost that grows with
// K while the store time it hides does not, so at larger K the single wide
// tile stays ahead.
//
// Operands and pipeline:
//  - The operands of one BK = 128 deep k stage stream through a 3-slot LDS
//    ring: A (q, int8 [M][K]) as BM rows of 128 bytes, B as 8 rows of BN
//    packed words.  The global->LDS copies are LDS-DMA buffer loads (the data
//    goes from the memory pipeline straight into LDS, not through registers).
//  - The copies of a stage are issued one per group of MFMAs through the step
//    that retires a slot, not in one burst: a burst of LDS-DMA instructions
//    from all waves at a barrier fills the vector memory queue, and a wave
//    stalled on a memory issue cannot issue its MFMAs.
//  - B stays packed until it reaches the registers: for a 16x16x64 MFMA lane
//    l supplies column l % 16 and the 16 k-values of group l / 16, which is
//    exactly one packed word Wpacked[j][n], expanded in registers into four
//    dwords of code bytes.  The words of the next k64 step are read one step
//    ahead, so the expansion never waits for LDS.
//  - Both operands are read through buffer resources, whose range check
//    returns zero past the end of the array (rows past M, chunks past K, word
//    rows past K/16) without touching memory.
//  - The MFMA takes the weights as its first operand and the activations as
//    its second, i.e. it computes the transposed tile: lane (g, l16) then ends
//    up with four consecutive output columns of one row, stored with one
//    16-byte write per 16 x 16 block.
//
// Tile order: workgroups are dealt round-robin to the 8 XCDs, each with its
// own L2, so the linear workgroup id is remapped to give every XCD a
// contiguous run of tiles, walked in groups of kGroupM tile rows; the tiles
// an XCD works on at once then share A rows and B columns in its L2.
#include "gemm_common.h"
#include "mmf_device.h"
#include "mmf_launch.h"

namespace mmf {
namespace {

// BX4: B rows are copied 16 bytes per lane (one word row per instruction),
// which needs N % 4 == 0 for aligned rows; otherwise 4 bytes per lane.
// The lane's index in its wave, computed afresh and hidden from the
// optimiser: values derived from it after a k loop that takes every register
// are then recomputed there instead of being kept (spilled) across the loop.
__device__ __forceinline__ int fresh_lane_id() {
  int l = static_cast<int>(__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)));
  asm volatile("" : "+v"(l));
  return l;
}

template <int BM, int BN, int WM, int WN, int BK, int S, bool BX4>
struct Tiling {
  static constexpr int kWavesM = BM / WM, kWavesN = BN / WN;
  static constexpr int kWaves = kWavesM * kWavesN;
  static constexpr int kThreads = kWaves * kWave;
  static constexpr int FM = WM / 16, FN = WN / 16;   // 16 x 16 MFMA tiles per wave
  static constexpr int KS = BK / 64;                 // k64 steps per stage
  static constexpr int kChunks = BK / 16;            // 16-byte chunks per A row
  // A stage: BM rows of BK bytes, unpadded (each LDS-DMA instruction writes
  // 1 KB contiguously), chunks XOR-swizzled per row against bank conflicts.
  static constexpr int kABytes = BM * BK;
  static constexpr int kAInstr = kABytes / 1024;
  // B stage: BK/16 word rows of BN words, each padded by 16 words so that the
  // four word rows one MFMA operand read spans fall on different banks.
  static constexpr int kBRow = BN + 16;
  static constexpr int kBBytes = (BK / 16) * kBRow * 4;
  static constexpr int kBInstr = BX4 ? (BK / 16) * BN / 256 : (BK / 16) * BN / 64;
  static constexpr int kAPerWave = kAInstr / kWaves, kBPerWave = kBInstr / kWaves;
  static constexpr int kLoadsPerStage = kAPerWave + kBPerWave;
  static constexpr int kStageBytes = kABytes + kBBytes;
  static_assert(kAInstr % kWaves == 0 && kBInstr % kWaves == 0, "loads must split evenly");
  static_assert(S == 3, "the stage waits below assume a 3-slot ring");
  static_assert(FN == 4 && FM >= 2, "expansion schedule: four words behind the fragment groups");
  static_assert(kLoadsPerStage <= FM, "one stage load per fragment group");
  static_assert(BK == 128, "A swizzle is for 8 chunks per row");
};

// Two waves per SIMD whatever the workgroup size: a 4-wave workgroup left to
// itself would take up to 512 registers per lane and keep a second workgroup
// off its CU.
template <int BM, int BN, int WM, int WN, int BK, int S, bool BX4, Epilogue EP>
__global__ __launch_bounds__((Tiling<BM, BN, WM, WN, BK, S, BX4>::kThreads))
__attribute__((amdgpu_waves_per_eu(2))) void gemm_kernel(
    const int8_t* __restrict__ q, const float* __restrict__ a_scale,
    const int32_t* __restrict__ q_rowsum, const uint32_t* __restrict__ Wp,
    const float* __restrict__ w_scale, void* __restrict__ out, int M, int K, int N, const Affine aff) {
  using T = Tiling<BM, BN, WM, WN, BK, S, BX4>;
  constexpr int FM = T::FM, FN = T::FN, KS = T::KS;
  // S ring slots, then the tile's per-row dequantisation factors
  __shared__ __attribute__((aligned(16))) char smem[S * T::kStageBytes + 8 * BM];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / T::kWavesN, wn = wave % T::kWavesN;
  const int l16 = lane & 15;
  const int g = lane >> 4;  // k group of this lane inside one MFMA
  int64_t tm, tn;
  tile_coords(blockIdx.x, (M + BM - 1) / BM, (N + BN - 1) / BN, tm, tn);
  const int m0 = static_cast<int>(tm) * BM;
  const int n0 = static_cast<int>(tn) * BN;
  const int J = K / 16;
  const int KT = (K + BK - 1) / BK;

  // Per-lane source offsets of this wave's LDS-DMA loads (k0 added per stage).
  // A instruction i covers rows 8 (wave * kAPerWave + i) .. + 7; the lane's
  // LDS slot s holds the row's logical chunk s ^ swz(row).  Instruction i + 2
  // reads the rows 16 below instruction i's, and the swizzle repeats every 16
  // rows, so only the first two instructions' offsets are kept (16 K is added
  // per pair after them): with four A loads per wave, four kept offsets push
  // the register count past 256 and spill inside the k loop.
  constexpr int kRowsPerInstr = 1024 / BK;
  static_assert(kRowsPerInstr == 8, "two A loads per 16-row swizzle period");
  constexpr int kA2 = T::kAPerWave < 2 ? T::kAPerWave : 2;
  uint32_t a_src[kA2];
  int a_chunk[kA2];
  // B instruction i: word row jj, a 256-word (BX4) or 64-word chunk of this
  // tile's columns.  Columns past N read the next word row or zero; their
  // outputs are dropped.
  uint32_t b_src[T::kBPerWave];
  int b_jj[T::kBPerWave], b_dst[T::kBPerWave];
  // The 4-wave tile's k loop takes all 256 registers.  There the offsets are
  // set from the lane index by set_offsets, again from a fresh lane index for
  // the stages after the last whole period, and the epilogue derives its
  // lane coordinates afresh too, so that nothing lane-derived is kept
  // (spilled) across the loop.  The 8-wave tiles set the same offsets inline
  // once, the form the register allocator handles best for them (through
  // set_offsets, without the second call, they spill).
  constexpr bool kFreshLane = T::kWaves == 4;
  static_assert(!kFreshLane || BX4, "the 4-wave tile copies B 16 bytes per lane");
  auto set_offsets = [&](int ln) {
#pragma unroll
    for (int i = 0; i < kA2; ++i) {
      const int r = (wave * T::kAPerWave + i) * kRowsPerInstr + ln / T::kChunks;
      const int c = (ln % T::kChunks) ^ a_swz(r);
      a_chunk[i] = c * 16;
      a_src[i] = static_cast<uint32_t>(m0 + r) * static_cast<uint32_t>(K) + static_cast<uint32_t>(c * 16);
    }
#pragma unroll
    for (int i = 0; i < T::kBPerWave; ++i) {
      const int idx = wave * T::kBPerWave + i;
      const int jj = idx / (BN / 256), q256 = idx % (BN / 256);
      b_jj[i] = jj;
      b_dst[i] = jj * T::kBRow * 4 + q256 * 1024;
      b_src[i] = 4u * (static_cast<uint32_t>(jj) * static_cast<uint32_t>(N) +
                       static_cast<uint32_t>(n0 + q256 * 256 + 4 * ln));
    }
  };
  if constexpr (kFreshLane) {
    set_offsets(lane);
  } else {
#pragma unroll
    for (int i = 0; i < kA2; ++i) {
      const int r = (wave * T::kAPerWave + i) * kRowsPerInstr + lane / T::kChunks;
      const int c = (lane % T::kChunks) ^ a_swz(r);
      a_chunk[i] = c * 16;
      a_src[i] = static_cast<uint32_t>(m0 + r) * static_cast<uint32_t>(K) + static_cast<uint32_t>(c * 16);
    }
#pragma unroll
    for (int i = 0; i < T::kBPerWave; ++i) {
      const int idx = wave * T::kBPerWave + i;
      if constexpr (BX4) {
        const int jj = idx / (BN / 256), q256 = idx % (BN / 256);
        b_jj[i] = jj;
        b_dst[i] = jj * T::kBRow * 4 + q256 * 1024;
        b_src[i] = 4u * (static_cast<uint32_t>(jj) * static_cast<uint32_t>(N) +
                         static_cast<uint32_t>(n0 + q256 * 256 + 4 * lane));
      } else {
        const int jj = idx / (BN / 64), q64 = idx % (BN / 64);
        b_jj[i] = jj;
        b_dst[i] = jj * T::kBRow * 4 + q64 * 256;
        b_src[i] = 4u * (static_cast<uint32_t>(jj) * static_cast<uint32_t>(N) +
                         static_cast<uint32_t>(n0 + q64 * 64 + lane));
      }
    }
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

  // Load i of stage kt into ring slot kt % S (i < kAPerWave: an A load, else
  // a B load).  The LDS-DMA loads are written as inline assembly, so the
  // compiler does not see LDS writes that could alias its fragment reads (it
  // would wait for every load in flight before each read); this kernel orders
  // them itself with explicit vmcnt waits before its barriers.  Offsets at or
  // past the end of a buffer (rows past M, chunks past K, word rows past
  // K/16, stages past the last) read zero without touching memory.
  auto issue_one = [&](int kt, int slot, int i) {
    const uint32_t base = lds0 + static_cast<uint32_t>(slot * T::kStageBytes);
    const int k0 = kt * BK;
    if (i < T::kAPerWave) {
      const uint32_t off = (k0 + a_chunk[i & 1] < K)
                               ? a_src[i & 1] + static_cast<uint32_t>(k0) +
                                     static_cast<uint32_t>((i >> 1) * 16) * static_cast<uint32_t>(K)
                               : 0x80000000u;
      const uint32_t dst = __builtin_amdgcn_readfirstlane(base + (wave * T::kAPerWave + i) * 1024);
      asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                   :
                   : "s"(dst), "v"(off), "s"(adesc)
                   : "memory", "m0");
    } else {
      const int b = i - T::kAPerWave;
      const int j0 = k0 / 16;
      const uint32_t off = (j0 + b_jj[b] < J) ? b_src[b] + static_cast<uint32_t>(j0) * b_row : 0x80000000u;
      const uint32_t dst = __builtin_amdgcn_readfirstlane(base + T::kABytes + b_dst[b]);
      if constexpr (BX4)
        asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                     :
                     : "s"(dst), "v"(off), "s"(bdesc)
                     : "memory", "m0");
      else
        asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, 0 offen lds"
                     :
                     : "s"(dst), "v"(off), "s"(bdesc)
                     : "memory", "m0");
    }
  };

  v4i acc[FM][FN];
#pragma unroll
  for (int a = 0; a < FM; ++a)
#pragma unroll
    for (int b = 0; b < FN; ++b) acc[a][b] = v4i{0, 0, 0, 0};

  // Fragments: A (16 rows x 64 k per lane group) refilled fragment by
  // fragment after each fragment's last use in the step; raw B words of the
  // next step; expanded code dwords of the current and the next step.
  v4i af[FM];
  uint32_t bw[FN];
  v4i be[2][FN];
  auto a_read = [&](int slot, int ks, int fm) -> v4i {
    const char* st = smem + slot * T::kStageBytes;
    const int row = wm * WM + fm * 16 + l16;
    const int c = (ks * 4 + g) ^ a_swz(row);
    return *reinterpret_cast<const v4i*>(st + row * BK + c * 16);
  };
  auto b_read = [&](int slot, int ks, int f) -> uint32_t {
    const uint32_t* Bs = reinterpret_cast<const uint32_t*>(smem + slot * T::kStageBytes + T::kABytes);
    return Bs[(ks * 4 + g) * T::kBRow + wn * WN + f * 16 + l16];
  };
  constexpr auto exp_lo = [](int fm) constexpr -> int {
    if constexpr (FM >= 2 * FN) return fm >= FM - FN ? fm - (FM - FN) : 0;
    else return fm == 0 ? 0 : ((fm - 1) * FN) / (FM - 1);
  };
  constexpr auto exp_hi = [](int fm) constexpr -> int {
    if constexpr (FM >= 2 * FN) return fm >= FM - FN ? fm - (FM - FN) + 1 : 0;
    else return fm == 0 ? 0 : (fm * FN) / (FM - 1);
  };
  auto expand = [](uint32_t x) -> v4i {
    return v4i{static_cast<int>(codes4(x, 0)), static_cast<int>(codes4(x, 1)),
               static_cast<int>(codes4(x, 2)), static_cast<int>(codes4(x, 3))};
  };

  // The tile's per-row dequantisation inputs (q_rowsum, then a_scale) go
  // into LDS by LDS-DMA too, one 64-row chunk per wave (2 BM / 64 waves), ahead of the ring's
  // first stages, so the prologue's wait covers them and the epilogue finds
  // them there.  Rows past M read zero.
  if (wave < 2 * BM / 64) {  // wave-uniform
    static_assert(2 * BM <= 64 * T::kWaves, "one row-factor chunk per wave");
    const int arr = wave / (BM / 64), chunk = wave % (BM / 64);
    const int row = m0 + chunk * 64 + lane;
    const uint32_t off = row < M ? 4u * static_cast<uint32_t>(row) : 0x80000000u;
    const uint64_t base = arr == 0 ? reinterpret_cast<uint64_t>(q_rowsum) : reinterpret_cast<uint64_t>(a_scale);
    const int bytes = (arr == 0 || EP != Epilogue::kRawI32) ? M * 4 : 0;
    const v4i desc = {static_cast<int>(static_cast<uint32_t>(base)), static_cast<int>((base >> 32) & 0xFFFF),
                      bytes, kBufferFlags};
    const uint32_t dst = __builtin_amdgcn_readfirstlane(
        lds0 + static_cast<uint32_t>(S * T::kStageBytes + arr * BM * 4 + chunk * 256));
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, 0 offen lds"
                 :
                 : "s"(dst), "v"(off), "s"(desc)
                 : "memory", "m0");
  }
  // Paired tiles with the GLU epilogue: the k loop's waves issue ahead of the
  // other workgroup's epilogue on the same SIMD (its SiLU arithmetic and
  // direct stores), which keeps the matrix cores fed (glu_gate 4-5 % faster;
  // the dequantising epilogue measured level and keeps the default).
  constexpr bool kLoopPriority = T::kWaves == 4 && EP == Epilogue::kGluF32;
  if constexpr (kLoopPriority) __builtin_amdgcn_s_setprio(1);
  // Prologue: stages 0 .. S-2, wait for stage 0 (and the row factors).
#pragma unroll
  for (int p = 0; p < S - 1; ++p)
#pragma unroll
    for (int i = 0; i < T::kLoadsPerStage; ++i) issue_one(p, p, i);
  __builtin_amdgcn_s_waitcnt(MMF_WAIT_VM((S - 2) * T::kLoadsPerStage));
  __builtin_amdgcn_s_barrier();
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) af[fm] = a_read(0, 0, fm);
#pragma unroll
  for (int f = 0; f < FN; ++f) bw[f] = b_read(0, 0, f);
#pragma unroll
  for (int f = 0; f < FN; ++f) be[0][f] = expand(bw[f]);

  // One k64 step (ks of stage kt, in ring slot `slot`; the next stage in
  // `slot_next`): the MFMAs of the step, the fragment reads of the next step
  // and the expansion of its words.  The last step of a stage reads the next
  // stage: it first waits for its own loads of that stage (with S = 3
  // nothing younger is in flight) and passes a barrier, which makes every
  // wave's loads visible and certifies that every wave has consumed the
  // oldest slot (its data fed MFMAs of earlier steps); that slot is then
  // refilled with stage kt + S - 1, one load per fragment group.
  auto step = [&](int kt, int ks, int slot, int slot_next, v4i (&bc)[FN], v4i (&bn)[FN]) {
    const bool refill = (ks == KS - 1);
    const int rslot = refill ? slot_next : slot, rks = refill ? 0 : ks + 1;
    __builtin_amdgcn_sched_barrier(0);
    if (refill) {
      __builtin_amdgcn_s_waitcnt(MMF_WAIT_VM((S - 3) * T::kLoadsPerStage));
      __builtin_amdgcn_s_barrier();
    }
#pragma unroll
    for (int f = 0; f < FN; ++f) bw[f] = b_read(rslot, rks, f);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
#pragma unroll
      for (int f = 0; f < FN; ++f)
        acc[fm][f] = __builtin_amdgcn_mfma_i32_16x16x64_i8(bc[f], af[fm], acc[fm][f], 0, 0, 0);
      af[fm] = a_read(rslot, rks, fm);
      if (refill && fm < T::kLoadsPerStage) issue_one(kt + S - 1, (slot + S - 1) % S, fm);
      // the next step's words, expanded behind this step's groups: one in
      // each of the last FN groups when there are at least 2 FN groups, else
      // spread over groups 1 .. FM - 1 (group 0 leaves their LDS reads time)
#pragma unroll
      for (int f = exp_lo(fm); f < exp_hi(fm); ++f) bn[f] = expand(bw[f]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // Whole periods of the ring (S stages) with every slot a compile-time
  // constant, so that LDS addresses are base + immediate and the loop's
  // back-edge, where the compiler's count of LDS reads in flight starts
  // over, comes once per S stages; then the remaining stages.  KS is even,
  // so a step's parity (which expanded-word buffer it reads) is ks's.
  static_assert(KS % 2 == 0, "step parity");
  int kt = 0;
  for (; kt + S <= KT; kt += S) {
#pragma unroll
    for (int j = 0; j < S; ++j)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) step(kt + j, ks, j, (j + 1) % S, be[ks % 2], be[(ks + 1) % 2]);
  }
  if constexpr (kFreshLane) {
    if (kt < KT) set_offsets(fresh_lane_id());
  }
  for (; kt < KT; ++kt) {
    const int slot = kt % S;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) step(kt, ks, slot, (slot + 1) % S, be[ks % 2], be[(ks + 1) % 2]);
  }
  if constexpr (kLoopPriority) __builtin_amdgcn_s_setprio(0);
  // no LDS-DMA write may still be in flight when the workgroup's LDS is freed
  __builtin_amdgcn_s_waitcnt(MMF_WAIT_VM_LGKM0(0));

  // ---- epilogue: the MFMA computed the transposed product, so lane
  // (g, l16) holds row l16 and columns 4 g .. 4 g + 3 of each 16 x 16 block ----
  const int elane = kFreshLane ? fresh_lane_id() : lane;
  const int el16 = elane & 15, eg = elane >> 4;
  const int* s_rsum = reinterpret_cast<const int*>(smem + S * T::kStageBytes);
  const float* s_scale = reinterpret_cast<const float*>(smem + S * T::kStageBytes + 4 * BM);
  const float ws = (EP == Epilogue::kDequantF32 || EP == Epilogue::kGluF32) ? w_scale[0] : 0.0f;
  const float ws_u = (EP == Epilogue::kGluF32) ? w_scale[1] : 0.0f;
  __syncthreads();
  constexpr uint32_t kOut = kOutOfRange;
  // affine epilogue: bias, lower bound, scale and activation of the lane's
  // four columns in each 16-column block (N % 16 == 0, one segment per block)
  ColAffine4 cf[FN];
  if constexpr (EP == Epilogue::kAffineF32) {
    static_assert(BX4, "affine output needs N % 4 == 0");
#pragma unroll
    for (int f = 0; f < FN; ++f) {
      const int n = n0 + wn * WN + f * 16 + 4 * eg;
      cf[f] = load_col_affine4(aff, w_scale, static_cast<uint32_t>(N), n < N ? static_cast<uint32_t>(n) : 0u);
    }
  }
  // The lane's four outputs of block (fm, f) (for the GLU, f is the gate/up
  // pair index: blocks 2f and 2f + 1 hold the same 16 channels, and lane
  // (g, l16) has channels 4 g .. 4 g + 3 of both).
  auto outputs = [&](int fm, int f) -> v4i {
    const int lr = wm * WM + fm * 16 + el16;
    const int rs = s_rsum[lr];
    v4i v;
    if constexpr (EP == Epilogue::kGluF32) {
      const float sg = s_scale[lr] * ws, su = s_scale[lr] * ws_u;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float gv = static_cast<float>(acc[fm][2 * f][r] - rs) * sg;
        const float uv = static_cast<float>(acc[fm][2 * f + 1][r] - rs) * su;
        v[r] = __float_as_int(gv * sigmoid_hw(gv) * uv);
      }
    } else {
      const float sc = s_scale[lr] * ws;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int d = acc[fm][f][r] - rs;
        if constexpr (EP == Epilogue::kAffineF32) {
          const float z = static_cast<float>(d) * (s_scale[lr] * cf[f].ws) + cf[f].bias[r];
          v[r] = __float_as_int(affine_act(z, cf[f].act, cf[f].lb[r]));
        } else {
          v[r] = (EP == Epilogue::kDequantF32) ? __float_as_int(static_cast<float>(d) * sc) : d;
        }
      }
    }
    return v;
  };
  constexpr bool kGlu = EP == Epilogue::kGluF32;
  // Plain outputs (dequantised or raw int32) leave through LDS as whole row
  // segments (below); the GLU and affine epilogues, whose output rows are
  // half as wide or whose launches are a single round, measured no faster
  // that way and keep direct 16-byte stores, and N % 4 != 0 takes
  // per-element stores.
  constexpr bool kStaged = BX4 && (EP == Epilogue::kDequantF32 || EP == Epilogue::kRawI32);
  if constexpr (!kStaged) {
    const int ow = kGlu ? N / 2 : N;  // output row length
    const uint32_t out_bytes = static_cast<uint32_t>(M) * static_cast<uint32_t>(ow) * 4u;
    const __amdgpu_buffer_rsrc_t orsrc =
        __builtin_amdgcn_make_buffer_rsrc(out, 0, static_cast<int>(out_bytes), kBufferFlags);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const int lr = wm * WM + fm * 16 + el16;
      const bool row_ok = m0 + lr < M;
      const uint32_t row_bytes = static_cast<uint32_t>(m0 + lr) * static_cast<uint32_t>(ow) * 4u;
#pragma unroll
      for (int f = 0; f < (kGlu ? FN / 2 : FN); ++f) {
        const int n = (kGlu ? (n0 + wn * WN) / 2 : n0 + wn * WN) + f * 16 + 4 * eg;
        const v4i v = outputs(fm, f);
        if constexpr (BX4) {
          // N % 4 == 0 (and L % 16 == 0): the four columns are all inside or all past the row
          const uint32_t off = (row_ok && n < ow) ? row_bytes + 4u * static_cast<uint32_t>(n) : kOut;
          __builtin_amdgcn_raw_buffer_store_b128(v, orsrc, off, 0, 0);
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const uint32_t off = (row_ok && n + r < N) ? row_bytes + 4u * static_cast<uint32_t>(n + r) : kOut;
            __builtin_amdgcn_raw_buffer_store_b32(static_cast<uint32_t>(v[r]), orsrc, off, 0, 0);
          }
        }
      }
    }
  } else {
    // Each wave's outputs leave through a private LDS buffer (the ring is
    // free now), 16 rows at a time: the wave writes its 16 x WN block as it
    // holds it (lane (g, l16): row l16, four columns of each 16-column block)
    // and reads it back as four store instructions of 4 rows x WN columns,
    // each row a contiguous 4 WN-byte segment.  Only the wave itself touches
    // its buffer, so no workgroup barrier is needed, and one buffer serves
    // every group of 16 rows: a wave's LDS operations are processed in issue
    // order, so the next group's writes land after this group's reads.  Rows
    // past M and columns past N fall outside the buffer's range or are sent
    // there explicitly.
    static_assert(WN == 64 && FN == 4, "a wave's row segment is 64 columns");
    constexpr int kRowB = WN * 4 + 16;       // staged row, padded by 16 bytes
    constexpr int kBufB = 16 * kRowB;
    static_assert(kBufB * T::kWaves <= S * T::kStageBytes, "a buffer per wave fits the ring");
    const int ow = N;
    const uint32_t out_bytes = static_cast<uint32_t>(M) * static_cast<uint32_t>(ow) * 4u;
    const __amdgpu_buffer_rsrc_t orsrc =
        __builtin_amdgcn_make_buffer_rsrc(out, 0, static_cast<int>(out_bytes), kBufferFlags);
    char* const buf = smem + wave * kBufB;
    const int rr = elane >> 4, qq = elane & 15;  // read-back lane: row rr of 4, column quad qq
    const int n = n0 + wn * WN + 4 * qq;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
#pragma unroll
      for (int f = 0; f < FN; ++f)
        *reinterpret_cast<v4i*>(buf + el16 * kRowB + (f * 16 + 4 * eg) * 4) = outputs(fm, f);
      // the wave's own writes, complete before it reads them back
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
      __builtin_amdgcn_s_waitcnt(MMF_WAIT_LGKM0);
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const v4i v = *reinterpret_cast<const v4i*>(buf + (4 * i + rr) * kRowB + qq * 16);
        const int m = m0 + wm * WM + fm * 16 + 4 * i + rr;
        const uint32_t off =
            (m < M && n < ow) ? (static_cast<uint32_t>(m) * static_cast<uint32_t>(ow) + static_cast<uint32_t>(n)) * 4u
                              : kOut;
        __builtin_amdgcn_raw_buffer_store_b128(v, orsrc, off, 0, 0);
      }
    }
  }
}

template <int BM, int BN, int WM, int WN, int BK, int S, bool BX4>
hipError_t launch_cfg(const ContractArgs& a, int64_t m_begin, int64_t m_rows, hipStream_t stream) {
  using T = Tiling<BM, BN, WM, WN, BK, S, BX4>;
  const int64_t gm = (m_rows + BM - 1) / BM;
  const int64_t gn = (a.N + BN - 1) / BN;
  const dim3 grid(static_cast<unsigned>(gm * gn));
  const dim3 block(T::kThreads);
  const int8_t* q = a.q + m_begin * a.K;
  const float* as = a.a_scale ? a.a_scale + m_begin : nullptr;
  const int32_t* rs = a.q_rowsum + m_begin;
  if (a.epilogue == Epilogue::kDequantF32)
    hipLaunchKernelGGL((gemm_kernel<BM, BN, WM, WN, BK, S, BX4, Epilogue::kDequantF32>), grid, block, 0,
                       stream, q, as, rs, a.Wpacked, a.w_scale,
                       static_cast<void*>(static_cast<float*>(a.out) + m_begin * a.N),
                       static_cast<int>(m_rows), a.K, static_cast<int>(a.N), a.affine);
  else if (a.epilogue == Epilogue::kAffineF32) {
    // not built for the paired 128 x 256 tile, which launch_gemm does not use
    // for this epilogue
    if constexpr (BX4 && T::kWaves == 8)
      hipLaunchKernelGGL((gemm_kernel<BM, BN, WM, WN, BK, S, true, Epilogue::kAffineF32>), grid, block, 0,
                         stream, q, as, rs, a.Wpacked, a.w_scale,
                         static_cast<void*>(static_cast<float*>(a.out) + m_begin * a.N),
                         static_cast<int>(m_rows), a.K, static_cast<int>(a.N), a.affine);
    else
      return hipErrorInvalidValue;
  } else if (a.epilogue == Epilogue::kGluF32) {
    if constexpr (BX4)
      hipLaunchKernelGGL((gemm_kernel<BM, BN, WM, WN, BK, S, true, Epilogue::kGluF32>), grid, block, 0, stream,
                         q, as, rs, a.Wpacked, a.w_scale,
                         static_cast<void*>(static_cast<float*>(a.out) + m_begin * (a.N / 2)),
                         static_cast<int>(m_rows), a.K, static_cast<int>(a.N), a.affine);
    else
      return hipErrorInvalidValue;
  } else
    hipLaunchKernelGGL((gemm_kernel<BM, BN, WM, WN, BK, S, BX4, Epilogue::kRawI32>), grid, block, 0,
                       stream, q, as, rs, a.Wpacked, a.w_scale,
                       static_cast<void*>(static_cast<int32_t*>(a.out) + m_begin * a.N),
                       static_cast<int>(m_rows), a.K, static_cast<int>(a.N), a.affine);
  return hipGetLastError();
}

}  // namespace

// The wide tile's area as two 128 x 256 workgroups per CU up to this depth
// (measured at M = 8192-16384: level or faster at K = 1024-4096 with the
// dequantising and GLU epilogues, up to 1 % slower at K = 5120 with large N).
// The affine epilogue keeps the wide tile: its paired form needs more than
// 256 registers inside the k loop and measured 3 % slower on the MLGRU gate
// projection (2048 x 2048 x 6144).
constexpr int kPairedTileMaxK = 4096;

// Whether the wide tiles of a problem run as paired 128 x 256 workgroups.
// The pairs pay off once a CU has a next tile whose k loop can cover a
// finished tile's stores, i.e. beyond one round of wide tiles (measured
// 4-12 % faster at K = 1024-4096).  Within a single round they gain only at
// small K on a nearly full round (K = 2048 with 192-256 wide tiles: 1-5 %)
// and lose elsewhere (144 tiles at K = 1040: 5 % slower, 256 at K = 3072: 3 %).
static bool gemm_paired(int64_t rows, int64_t N, int K, int cus, Epilogue ep) {
  if (K > kPairedTileMaxK || ep == Epilogue::kAffineF32) return false;
  const int64_t c = cus > 0 ? cus : 256;
  const int64_t wide = ((rows + 127) / 128) * ((N + 511) / 512);
  return wide > c || (K <= 2048 && 4 * wide >= 3 * c);
}

int gemm_tile_choice(int64_t rows, int64_t N, int cus) {
  // Estimated time = rounds of workgroups over the CUs x the time of one
  // tile's k loop when it runs alone, measured relative to each other at
  // K = 2048 (128 x 512 : 64 x 512 : 64 x 256 = 29.5 : 18.6 : 14.0 us, i.e.
  // 21 : 13 : 10).  The widest tile has the most reuse per operand byte and
  // wins once a problem fills the CUs; a problem with few such tiles (short
  // M, or narrow N) finishes sooner with more, smaller tiles.  Ties keep the
  // wider tile.
  struct Shape { int64_t bm, bn, cost; };
  constexpr Shape kShapes[] = {{128, 512, 21}, {64, 512, 13}, {64, 256, 10}};
  const int64_t c = cus > 0 ? cus : 256;
  int best = 0;
  int64_t best_t = -1;
  for (int i = 0; i < 3; ++i) {
    const int64_t tiles = ((rows + kShapes[i].bm - 1) / kShapes[i].bm) * ((N + kShapes[i].bn - 1) / kShapes[i].bn);
    const int64_t t = (tiles + c - 1) / c * kShapes[i].cost;
    if (best_t < 0 || t < best_t) {
      best = i;
      best_t = t;
    }
  }
  return best;
}

int gemm_plan(int64_t rows, int K, int64_t N, Epilogue ep, int cus) {
  if (N % 4 != 0) return kPlan256x256;
  const int choice = gemm_tile_choice(rows, N, cus);
  if (choice == 1) return kPlan64x512;
  if (choice == 2) return kPlan64x256;
  return gemm_paired(rows, N, K, cus, ep) ? kPlan128x256Paired : kPlan128x512;
}

hipError_t launch_gemm(const ContractArgs& a, hipStream_t stream) {
  // 32-bit buffer offsets: a launch covers at most 2^31 - 1 bytes of q, of
  // packed weights and of output; taller problems run in row slices.  The
  // C-ABI layer rejects shapes without a slice before enqueueing anything.
  const int64_t slice = gemm_row_slice(a.K, a.N);
  if (slice == 0) return hipErrorInvalidValue;
  const int cus = device_cus();
  for (int64_t m0 = 0; m0 < a.M; m0 += slice) {
    const int64_t rows = a.M - m0 < slice ? a.M - m0 : slice;
    hipError_t e;
    switch (gemm_plan(rows, a.K, a.N, a.epilogue, cus)) {
      case kPlan256x256: e = launch_cfg<256, 256, 128, 64, 128, 3, false>(a, m0, rows, stream); break;
      case kPlan64x512: e = launch_cfg<64, 512, 64, 64, 128, 3, true>(a, m0, rows, stream); break;
      case kPlan64x256: e = launch_cfg<64, 256, 32, 64, 128, 3, true>(a, m0, rows, stream); break;
      case kPlan128x256Paired: e = launch_cfg<128, 256, 128, 64, 128, 3, true>(a, m0, rows, stream); break;
      default: e = launch_cfg<128, 512, 128, 64, 128, 3, true>(a, m0, rows, stream); break;
    }
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace mmf
