// Pieces shared by the tiled matrix-core kernels (the prefill contraction
// and the two backward products): the XCD-aware tile order, the waitcnt
// immediates of the hand-scheduled loops, the LDS chunk swizzle of 128-byte
// operand rows and the LDS-DMA load.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mmf {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int kBufferFlags = 0x00020000;  // gfx9 buffer descriptor word 3
constexpr int kXcds = 8;
constexpr int kGroupM = 4;
constexpr uint32_t kOutOfRange = 0x80000000u;  // a buffer offset past every range

// Tile order: workgroups are dealt round-robin to the 8 XCDs, each with its
// own L2, so the linear workgroup id b is remapped to give every XCD a
// contiguous run of tiles, walked in groups of kGroupM tile rows; the tiles
// an XCD works on at once then share operand rows and columns in its L2.
__device__ __forceinline__ void tile_coords(int64_t b, int64_t tiles_m, int64_t tiles_n, int64_t& tm,
                                            int64_t& tn) {
  const int64_t total = tiles_m * tiles_n;
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
// LDS / scalar memory counter only (vmcnt and expcnt at their maxima)
#define MMF_WAIT_LGKM0 (0xF | (0x7 << 4) | (0x3 << 14))

// Chunk swizzle of 128-byte LDS rows (8 chunks of 16 bytes per row): row r
// stores logical chunk c in slot c ^ swz(r).  Sixteen consecutive rows at one
// chunk then hit distinct bank groups both when 8 lanes share 32 banks and
// when 16 lanes share 64 banks; swz(r + 16) = swz(r).
__device__ __forceinline__ int a_swz(int r) { return ((r >> 1) ^ (r << 2)) & 7; }

__device__ __forceinline__ v4i buffer_desc(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  return v4i{static_cast<int>(static_cast<uint32_t>(a)), static_cast<int>((a >> 32) & 0xFFFF),
             static_cast<int>(bytes), kBufferFlags};
}

// LDS-DMA loads: 16 (dwordx4) or 4 bytes per lane from buffer offset `off`
// (zero past the range) straight into LDS at lds_dst + 16 lane (or 4 lane).
// Written as inline assembly, so the compiler sees no LDS write that could
// alias its own LDS reads; callers order them with explicit waits.
__device__ __forceinline__ void lds_dma16(uint32_t lds_dst, uint32_t off, v4i desc) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds_dst), "v"(off), "s"(desc)
               : "memory", "m0");
}
__device__ __forceinline__ void lds_dma4(uint32_t lds_dst, uint32_t off, v4i desc) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, 0 offen lds"
               :
               : "s"(lds_dst), "v"(off), "s"(desc)
               : "memory", "m0");
}

}  // namespace mmf
