// MLGRU recurrence and output gate (Sec. "MatMul-free Language Model
// Architecture", MLGRU equations):
//   h_t  = f_t (.) h_{t-1} + (1 - f_t) (.) c_t
//   o'_t = g_t (.) sigmoid(h_t)
// over B sequences of T tokens, the gates f, c, g coming side by side in the
// rows of fcg [B*T][3d] as the projection kernels write them.
//
// The recurrence is linear in h, so a chunk of L tokens maps the state that
// enters it to A h + B, with A the product of its forget gates and B the
// state it ends in from h = 0.  Long sequences therefore run as three
// launches: (1) A and B of every chunk and channel; (2) for every channel,
// the state entering each chunk, composed over the chunks in order;
// (3) every chunk again from its entering state, writing o' and, in the last
// chunk, the final state.  A sequence of at most L tokens is one launch of
// (3) from h_0.  All work is streaming: one thread holds four adjacent
// channels, so each wave reads 1 KB contiguous per array and token, and the
// loads of the next tokens are in flight while the state is updated.
#include "mmf_device.h"
#include "mmf_launch.h"

namespace mmf {
namespace {

constexpr int kBlock = 256;
constexpr int kUnroll = 8;       // tokens whose loads are in flight together
constexpr int kCarryCh = 32;     // channels per workgroup of the carry pass
constexpr int64_t kMinChunk = 16;
constexpr int64_t kMaxChunks = 128;

__device__ __forceinline__ float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ void st4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }


struct ChunkIdx {
  int64_t b, k, i;  // sequence, chunk, first channel (multiple of 4)
};
__device__ __forceinline__ ChunkIdx chunk_idx(int64_t idx, int64_t nchunk, int64_t d) {
  const int64_t d4 = d / 4;
  const int64_t bk = idx / d4;
  return {bk / nchunk, bk % nchunk, 4 * (idx % d4)};
}

// (1) A = prod f and B = the chunk's state from h = 0, per chunk and channel.
__global__ __launch_bounds__(kBlock) void mlgru_chunk_kernel(const float* __restrict__ fcg, int64_t T, int64_t d,
                                                             int64_t L, int64_t nchunk, int64_t total,
                                                             float* __restrict__ A, float* __restrict__ Bs) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (idx >= total) return;
  const ChunkIdx ci = chunk_idx(idx, nchunk, d);
  const int64_t t0 = ci.k * L;
  const int64_t t1 = t0 + L < T ? t0 + L : T;
  const float* base = fcg + (ci.b * T) * 3 * d + ci.i;
  float4 a = {1.0f, 1.0f, 1.0f, 1.0f}, h = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int64_t t = t0; t < t1; t += kUnroll) {
    float4 fv[kUnroll], cv[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t tt = t + u < t1 ? t + u : t1 - 1;
      fv[u] = ld4(base + tt * 3 * d);
      cv[u] = ld4(base + tt * 3 * d + d);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (t + u < t1) {
        a.x *= fv[u].x; a.y *= fv[u].y; a.z *= fv[u].z; a.w *= fv[u].w;
        h.x = mlgru_step(h.x, fv[u].x, cv[u].x);
        h.y = mlgru_step(h.y, fv[u].y, cv[u].y);
        h.z = mlgru_step(h.z, fv[u].z, cv[u].z);
        h.w = mlgru_step(h.w, fv[u].w, cv[u].w);
      }
    }
  }
  const int64_t o = (ci.b * nchunk + ci.k) * d + ci.i;
  st4(A + o, a);
  st4(Bs + o, h);
}

// (2) state entering each chunk: h <- A_k h + B_k in chunk order.  A
// workgroup owns kCarryCh channels of one sequence.  Its threads first copy
// the summaries of every chunk into LDS (all loads issued before any store),
// then each of kSegs groups composes a run of consecutive chunks into one
// map h -> a h + b, one group joins the kSegs maps in order, and each group
// walks its run again from the state entering it, writing the carries: the
// chain of dependent steps is 2 nchunk / kSegs + kSegs long, not nchunk.
__global__ __launch_bounds__(kBlock) void mlgru_carry_kernel(const float* __restrict__ A,
                                                             const float* __restrict__ Bs,
                                                             const float* __restrict__ h0, int64_t nchunk,
                                                             int64_t d, float* __restrict__ carry) {
  constexpr int kSegs = kBlock / kCarryCh;
  constexpr int kPerThread = kMaxChunks * kCarryCh / kBlock;
  __shared__ float sa[kMaxChunks][kCarryCh];
  __shared__ float sb[kMaxChunks][kCarryCh];
  __shared__ float seg_a[kSegs][kCarryCh], seg_b[kSegs][kCarryCh], seg_h[kSegs][kCarryCh];
  const int64_t nblk = (d + kCarryCh - 1) / kCarryCh;
  const int64_t b = blockIdx.x / nblk;
  const int64_t c0 = (blockIdx.x % nblk) * kCarryCh;
  const int nch = static_cast<int>(nchunk);
  const int64_t base = b * nchunk * d + c0;
  const int c = threadIdx.x % kCarryCh, sg = threadIdx.x / kCarryCh;
  const bool col_ok = c0 + c < d;
  {
    float ra[kPerThread], rb[kPerThread];
#pragma unroll
    for (int u = 0; u < kPerThread; ++u) {
      const int k = sg + kSegs * u;  // element threadIdx.x + kBlock u
      const bool ok = col_ok && k < nch;
      ra[u] = ok ? A[base + k * d + c] : 1.0f;
      rb[u] = ok ? Bs[base + k * d + c] : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < kPerThread; ++u) {
      sa[sg + kSegs * u][c] = ra[u];
      sb[sg + kSegs * u][c] = rb[u];
    }
  }
  __syncthreads();
  const int per = (nch + kSegs - 1) / kSegs;
  const int k0 = sg * per < nch ? sg * per : nch;
  const int k1 = k0 + per < nch ? k0 + per : nch;
  float ca = 1.0f, cb = 0.0f;  // composed map of the run [k0, k1)
  for (int k = k0; k < k1; ++k) {
    ca = sa[k][c] * ca;
    cb = sa[k][c] * cb + sb[k][c];
  }
  seg_a[sg][c] = ca;
  seg_b[sg][c] = cb;
  __syncthreads();
  if (sg == 0) {
    float h = (h0 != nullptr && col_ok) ? h0[b * d + c0 + c] : 0.0f;
#pragma unroll
    for (int s = 0; s < kSegs; ++s) {
      seg_h[s][c] = h;
      h = seg_a[s][c] * h + seg_b[s][c];
    }
  }
  __syncthreads();
  if (!col_ok) return;
  float h = seg_h[sg][c];
  for (int k = k0; k < k1; ++k) {
    carry[base + k * d + c] = h;
    h = sa[k][c] * h + sb[k][c];
  }
}

// (3) the recurrence of each chunk from its entering state, with the output
// gate; the last chunk of a sequence stores the final state.
__global__ __launch_bounds__(kBlock) void mlgru_apply_kernel(const float* __restrict__ fcg,
                                                             const float* __restrict__ carry,
                                                             const float* h0, int64_t T, int64_t d, int64_t L,
                                                             int64_t nchunk, int64_t total, float* __restrict__ o,
                                                             float* h_last) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (idx >= total) return;
  const ChunkIdx ci = chunk_idx(idx, nchunk, d);
  const int64_t t0 = ci.k * L;
  const int64_t t1 = t0 + L < T ? t0 + L : T;
  float4 h;
  if (nchunk > 1)
    h = ld4(carry + (ci.b * nchunk + ci.k) * d + ci.i);
  else if (h0 != nullptr)
    h = ld4(h0 + ci.b * d + ci.i);
  else
    h = {0.0f, 0.0f, 0.0f, 0.0f};
  const float* base = fcg + (ci.b * T) * 3 * d + ci.i;
  float* obase = o + (ci.b * T) * d + ci.i;
  for (int64_t t = t0; t < t1; t += kUnroll) {
    float4 fv[kUnroll], cv[kUnroll], gv[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t tt = t + u < t1 ? t + u : t1 - 1;
      fv[u] = ld4(base + tt * 3 * d);
      cv[u] = ld4(base + tt * 3 * d + d);
      gv[u] = ld4(base + tt * 3 * d + 2 * d);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (t + u < t1) {
        h.x = mlgru_step(h.x, fv[u].x, cv[u].x);
        h.y = mlgru_step(h.y, fv[u].y, cv[u].y);
        h.z = mlgru_step(h.z, fv[u].z, cv[u].z);
        h.w = mlgru_step(h.w, fv[u].w, cv[u].w);
        const float4 ov = {mlgru_out_gate(gv[u].x, h.x), mlgru_out_gate(gv[u].y, h.y), mlgru_out_gate(gv[u].z, h.z),
                           mlgru_out_gate(gv[u].w, h.w)};
        st4(obase + (t + u) * d, ov);
      }
    }
  }
  if (ci.k == nchunk - 1 && h_last != nullptr) st4(h_last + ci.b * d + ci.i, h);
}

unsigned blocks_for(int64_t threads) { return static_cast<unsigned>((threads + kBlock - 1) / kBlock); }

}  // namespace

int64_t mlgru_chunk_len(int64_t B, int64_t T, int64_t d) {
  (void)B;
  (void)d;
  if (T <= kMinChunk) return T > 0 ? T : 1;
  const int64_t L = (T + kMaxChunks - 1) / kMaxChunks;
  return L < kMinChunk ? kMinChunk : L;
}

int64_t mlgru_scan_ws_floats(int64_t B, int64_t T, int64_t d) {
  const int64_t L = mlgru_chunk_len(B, T, d);
  const int64_t nchunk = (T + L - 1) / L;
  return nchunk > 1 ? 3 * B * nchunk * d : 0;
}

hipError_t launch_mlgru_scan(const float* fcg, const float* h0, float* o, float* h_last, int64_t B,
                             int64_t T, int64_t d, float* ws, hipStream_t stream) {
  if (B <= 0 || T <= 0 || d <= 0) return hipSuccess;
  if (d % 4 != 0) return hipErrorInvalidValue;
  const int64_t L = mlgru_chunk_len(B, T, d);
  const int64_t nchunk = (T + L - 1) / L;
  const int64_t total = B * nchunk * (d / 4);
  float* carry = nullptr;
  if (nchunk > 1) {
    if (ws == nullptr) return hipErrorInvalidValue;
    float* A = ws;
    float* Bs = ws + B * nchunk * d;
    carry = ws + 2 * B * nchunk * d;
    hipLaunchKernelGGL(mlgru_chunk_kernel, dim3(blocks_for(total)), dim3(kBlock), 0, stream, fcg, T, d, L,
                       nchunk, total, A, Bs);
    hipLaunchKernelGGL(mlgru_carry_kernel, dim3(static_cast<unsigned>(B * ((d + kCarryCh - 1) / kCarryCh))),
                       dim3(kBlock), 0, stream, A, Bs, h0, nchunk, d, carry);
  }
  hipLaunchKernelGGL(mlgru_apply_kernel, dim3(blocks_for(total)), dim3(kBlock), 0, stream, fcg, carry, h0, T, d,
                     L, nchunk, total, o, h_last);
  return hipGetLastError();
}

}  // namespace mmf
