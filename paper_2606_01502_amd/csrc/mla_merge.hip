// Log-sum-exp merge of partial attention outputs (the requester's online
// softmax recombination, paper Sections 2.2, 3.3 and 4.2), and the split-K
// combine that applies the same algebra to one job's slot-range partials.
//
// Per row, over the live parts (lse != -inf):
//   L = max lse_j,  lse = L + ln sum exp(lse_j - L),  out = sum exp(lse_j - lse) o_j.
// A part with lse = -inf is skipped (its o is never read, so a NaN there
// cannot leak); no live part gives out = 0, lse = -inf.
//
// HBM-bound elementwise work: 128 lanes per 512-wide row, each lane moving
// 16-byte vectors; every lane of a row recomputes the row's weights from the
// n lse values (a few exp per lane against n 16-byte loads).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mla_kernels.h"

namespace mla {
namespace {

typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kRowsPerBlock = kThreads / 128;  // 2 rows of 512 floats per workgroup

// Merged lse of one row's parts; -inf when no part is live.
template <typename LseAt>
__device__ __forceinline__ float merged_lse(int n, LseAt lse_at) {
  float m = -INFINITY;
  for (int j = 0; j < n; ++j) m = fmaxf(m, lse_at(j));
  if (m == -INFINITY) return -INFINITY;
  float s = 0.f;
  for (int j = 0; j < n; ++j) {
    const float l = lse_at(j);
    if (l != -INFINITY) s += __expf(l - m);
  }
  return m + __logf(s);
}

// sum over live parts of exp(lse_j - lse) * o_j[col .. col+3]
template <typename LseAt, typename RowAt>
__device__ __forceinline__ f32x4_t merged_row(int n, float lse, LseAt lse_at, RowAt row_at) {
  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
  if (lse == -INFINITY) return acc;
  for (int j = 0; j < n; ++j) {
    const float l = lse_at(j);
    if (l != -INFINITY) acc += __expf(l - lse) * *row_at(j);
  }
  return acc;
}

__global__ __launch_bounds__(kThreads) void merge_kernel(const MergeParams p) {
  const int n_rows = p.B * p.Mq * p.H;
  const int row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 7);
  if (row >= n_rows) return;
  const int col = (threadIdx.x & 127) * 4;
  const int b = row / (p.Mq * p.H);
  const int rem = row - b * (p.Mq * p.H);
  const int i = rem / p.H, h = rem - (rem / p.H) * p.H;
  const int64_t lo = b * p.l_s0 + i * p.l_s1 + h * p.l_s2;
  const int64_t oo = b * p.o_s0 + i * p.o_s1 + h * p.o_s2 + col;
  auto lse_at = [&](int j) { return p.lse[j][lo]; };
  const float lse = merged_lse(p.n_parts, lse_at);
  const f32x4_t acc = merged_row(p.n_parts, lse, lse_at,
                                 [&](int j) { return (const f32x4_t*)(p.o[j] + oo); });
  *(f32x4_t*)(p.out + b * p.out_s0 + i * p.out_s1 + h * p.out_s2 + col) = acc;
  if (p.out_lse && col == 0) p.out_lse[b * p.ol_s0 + i * p.ol_s1 + h * p.ol_s2] = lse;
}

__global__ __launch_bounds__(kThreads) void combine_kernel(const CombineParams p) {
  const int n_rows = p.R * p.rows;
  const int grow = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 7);
  if (grow >= n_rows) return;
  const int col = (threadIdx.x & 127) * 4;
  const int r = grow / p.rows;
  const int row = grow - r * p.rows;
  const int64_t base = (int64_t)r * p.S * p.rows + row;  // split j of (r, row) at base + j*rows
  auto lse_at = [&](int j) { return p.ws_lse[base + (int64_t)j * p.rows]; };
  const float lse = merged_lse(p.S, lse_at);
  const f32x4_t acc = merged_row(p.S, lse, lse_at, [&](int j) {
    return (const f32x4_t*)(p.ws_o + (base + (int64_t)j * p.rows) * kDLat + col);
  });
  const int i = row / p.H, h = row - (row / p.H) * p.H;
  *(f32x4_t*)(p.out + r * p.out_s0 + i * p.out_s1 + h * p.out_s2 + col) = acc;
  if (col == 0) p.lse[r * p.lse_s0 + i * p.lse_s1 + h * p.lse_s2] = lse;
}

}  // namespace

hipError_t launch_merge(const MergeParams& p, hipStream_t s) {
  const int64_t n_rows = (int64_t)p.B * p.Mq * p.H;
  if (n_rows == 0) return hipSuccess;
  const int grid = (int)((n_rows + kRowsPerBlock - 1) / kRowsPerBlock);
  hipLaunchKernelGGL(merge_kernel, dim3(grid), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_combine(const CombineParams& p, hipStream_t s) {
  const int64_t n_rows = (int64_t)p.R * p.rows;
  if (n_rows == 0) return hipSuccess;
  const int grid = (int)((n_rows + kRowsPerBlock - 1) / kRowsPerBlock);
  hipLaunchKernelGGL(combine_kernel, dim3(grid), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace mla
