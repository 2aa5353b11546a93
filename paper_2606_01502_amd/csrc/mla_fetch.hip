// FETCH-side copies on one GPU (paper Section 2.2): the scattered gather of a
// selected token set into a contiguous payload, and the splice of a pulled
// chunk into the requester's paged pool with its RoPE part turned by a
// position offset.  Both are pure HBM streams: each workgroup moves 64 tokens
// of one layer, every 1 KiB latent row by 64 lanes with 16-byte accesses, and
// all layers of a chunk go out in one launch.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mla_kernels.h"

namespace mla {
namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// float -> bf16 bits, round to nearest even (finite inputs)
__device__ __forceinline__ uint32_t to_bf16(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ uint32_t pack(float lo, float hi) {
  return to_bf16(lo) | (to_bf16(hi) << 16);
}

// Rotate pair (x, y) by the angle whose cosine and sine are c, s.
__device__ __forceinline__ void turn(float& x, float& y, float c, float s) {
  const float nx = x * c - y * s;
  const float ny = x * s + y * c;
  x = nx;
  y = ny;
}

// Gather: out row j of layer l = pool token sel[j] (zero row for an empty or
// invalid slot).
__global__ __launch_bounds__(256) void gather_kernel(const FetchParams p) {
  const int64_t groups = (p.n + kBlock - 1) / kBlock;
  const int64_t l = blockIdx.x / groups;
  const int64_t j0 = (blockIdx.x - l * groups) * kBlock;
  const int tid = threadIdx.x;
  __shared__ int64_t src_row[kBlock];  // pool row of slot j0 + t, or -1
  if (tid < kBlock) {
    int64_t row = -1;
    const int64_t j = j0 + tid;
    if (j < p.n) {
      const int32_t s = p.sel[j];
      if (s >= 0 && s < p.n_ids) {
        const int32_t b = p.table[s / kBlock];
        if (b >= 0 && b < p.P) row = (l * p.P + b) * kBlock + (s % kBlock);
      }
    }
    src_row[tid] = row;
  }
  __syncthreads();
  const u32x4_t* sc = (const u32x4_t*)p.src_ckv;
  const u32x4_t* sk = (const u32x4_t*)p.src_kpe;
  u32x4_t* dc = (u32x4_t*)p.dst_ckv;
  u32x4_t* dk = (u32x4_t*)p.dst_kpe;
  // latent rows: 64 chunks of 16 B per token, 4 tokens per pass
#pragma unroll 4
  for (int it = 0; it < 16; ++it) {
    const int c = it * 256 + tid;
    const int t = c >> 6, col = c & 63;
    const int64_t j = j0 + t;
    if (j < p.n) {
      const int64_t row = src_row[t];
      const u32x4_t v = row >= 0 ? sc[row * 64 + col] : u32x4_t{0u, 0u, 0u, 0u};
      dc[(l * p.n + j) * 64 + col] = v;
    }
  }
  // RoPE rows: 8 chunks per token
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const int c = it * 256 + tid;
    const int t = c >> 3, col = c & 7;
    const int64_t j = j0 + t;
    if (j < p.n) {
      const int64_t row = src_row[t];
      const u32x4_t v = row >= 0 ? sk[row * 8 + col] : u32x4_t{0u, 0u, 0u, 0u};
      dk[(l * p.n + j) * 8 + col] = v;
    }
  }
}

// Splice: chunk token t of layer l goes to slot dst_start + t of the
// requester's sequence, its RoPE pairs turned by (cs, sn).  Tokens whose
// block-table entry is outside [0, P) are skipped.
__global__ __launch_bounds__(256) void splice_kernel(const FetchParams p) {
  const int64_t groups = (p.n + kBlock - 1) / kBlock;
  const int64_t l = blockIdx.x / groups;
  const int64_t t0 = (blockIdx.x - l * groups) * kBlock;
  const int tid = threadIdx.x;
  __shared__ int64_t dst_row[kBlock];  // pool row of chunk token t0 + t, or -1
  if (tid < kBlock) {
    int64_t row = -1;
    const int64_t t = t0 + tid;
    if (t < p.n) {
      const int64_t slot = p.dst_start + t;
      const int32_t b = p.table[slot / kBlock];
      if (b >= 0 && b < p.P) row = (l * p.P + b) * kBlock + (slot % kBlock);
    }
    dst_row[tid] = row;
  }
  __syncthreads();
  const u32x4_t* sc = (const u32x4_t*)p.src_ckv;
  const u32x4_t* sk = (const u32x4_t*)p.src_kpe;
  u32x4_t* dc = (u32x4_t*)p.dst_ckv;
  u32x4_t* dk = (u32x4_t*)p.dst_kpe;
#pragma unroll 4
  for (int it = 0; it < 16; ++it) {
    const int c = it * 256 + tid;
    const int t = c >> 6, col = c & 63;
    const int64_t row = dst_row[t];
    if (t0 + t < p.n && row >= 0) dc[row * 64 + col] = sc[(l * p.n + t0 + t) * 64 + col];
  }
  // RoPE: lane (t, q) takes chunks q and q + 4 of token t's row, dims
  // 8q .. 8q+7 and 8q+32 .. 8q+39, which hold whole pairs in both pairings
  const int t = tid >> 2, q = tid & 3;
  const int64_t row = dst_row[t];
  if (t0 + t < p.n && row >= 0) {
    const u32x4_t* src = sk + (l * p.n + t0 + t) * 8;
    const u32x4_t a = src[q], b = src[q + 4];
    float x[8], y[8];  // dims 8q + e and 8q + 32 + e
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      x[2 * k] = bf16_lo(a[k]);
      x[2 * k + 1] = bf16_hi(a[k]);
      y[2 * k] = bf16_lo(b[k]);
      y[2 * k + 1] = bf16_hi(b[k]);
    }
    if (p.pairing == 0) {
      // pairs (2i, 2i+1): i = 4q + k in the first chunk, 16 + 4q + k in the second
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        turn(x[2 * k], x[2 * k + 1], p.cs[4 * q + k], p.sn[4 * q + k]);
        turn(y[2 * k], y[2 * k + 1], p.cs[16 + 4 * q + k], p.sn[16 + 4 * q + k]);
      }
    } else {
      // pairs (i, i + 32): i = 8q + e
#pragma unroll
      for (int e = 0; e < 8; ++e) turn(x[e], y[e], p.cs[8 * q + e], p.sn[8 * q + e]);
    }
    u32x4_t oa, ob;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      oa[k] = pack(x[2 * k], x[2 * k + 1]);
      ob[k] = pack(y[2 * k], y[2 * k + 1]);
    }
    dk[row * 8 + q] = oa;
    dk[row * 8 + q + 4] = ob;
  }
}

}  // namespace

hipError_t launch_fetch_gather(const FetchParams& p, hipStream_t s) {
  const int64_t grid = (int64_t)p.L * ((p.n + kBlock - 1) / kBlock);
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL(gather_kernel, dim3((uint32_t)grid), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_fetch_splice(const FetchParams& p, hipStream_t s) {
  const int64_t grid = (int64_t)p.L * ((p.n + kBlock - 1) / kBlock);
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL(splice_kernel, dim3((uint32_t)grid), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace mla
