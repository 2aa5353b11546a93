// Log-sum-exp merge of partial attention outputs (the requester's online
// softmax recombination, paper Sections 2.2, 3.3 and 4.2), and the split-K
// combine that applies the same algebra to one job's slot-range partials.
// Both run the row routine of mla_rowmerge.h: HBM-bound, one wave per row.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mla_kernels.h"
#include "mla_rowmerge.h"

namespace mla {
namespace {

using namespace rowmerge;

constexpr int kRowsPerBlock = kThreads / 64;  // one wave per row

__global__ __launch_bounds__(kThreads) void merge_kernel(const MergeParams p) {
  const int n_rows = p.B * p.Mq * p.H;
  const int row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (row >= n_rows) return;
  const int lane = threadIdx.x & 63;
  const int b = row / (p.Mq * p.H);
  const int rem = row - b * (p.Mq * p.H);
  const int i = rem / p.H, h = rem - (rem / p.H) * p.H;
  const int64_t lo = b * p.l_s0 + i * p.l_s1 + h * p.l_s2;
  const int64_t oo = b * p.o_s0 + i * p.o_s1 + h * p.o_s2;
  f32x4_t acc0, acc1;
  float lse;
  if (p.wire) {
    // wire-form parts: lse = m + ln l from the (m, l) pair (-inf when l = 0)
    lse = merge_parts<true, Bf16Rows>(
        p.n_parts,
        [&](int j) {
          const float m = p.lse[j][lo], l = p.lse[j][lo + 1];
          return l > 0.f ? m + __logf(l) : -INFINITY;
        },
        [&](int j) { return (const uint16_t*)p.o[j] + oo; }, [](int) { return 1.f; }, acc0, acc1,
        lane);
  } else {
    lse = merge_parts<true, F32Rows>(
        p.n_parts, [&](int j) { return p.lse[j][lo]; },
        [&](int j) { return (const float*)p.o[j] + oo; }, [](int) { return 1.f; }, acc0, acc1, lane);
  }
  store_row(p.out + b * p.out_s0 + i * p.out_s1 + h * p.out_s2, acc0, acc1, lane);
  if (p.out_lse && lane == 0) p.out_lse[b * p.ol_s0 + i * p.ol_s1 + h * p.ol_s2] = lse;
}

__global__ __launch_bounds__(kThreads) void combine_kernel(const CombineParams p) {
  const int n_rows = p.R * p.rows;
  // renumbered like the partial kernel (each XCD a contiguous range), so that
  // a row tile's rows tend to be combined on the XCD whose L2 holds its
  // splits' rows
  const int blk = gridDim.x % 8 ? (int)blockIdx.x
                               : (int)(blockIdx.x % 8) * (int)(gridDim.x / 8) + (int)(blockIdx.x / 8);
  const int grow = blk * kRowsPerBlock + (threadIdx.x >> 6);
  if (grow >= n_rows) return;
  const int lane = threadIdx.x & 63;
  const int r = grow / p.rows;
  const int row = grow - r * p.rows;
  combine_row(p, p.S, r, row, lane);
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
