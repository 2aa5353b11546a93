// The row routines of the log-sum-exp merge (Sections 3.3 and 4.2) used by the
// merge and split-K combine kernels: one wave merges one row of n parts.
//
// Per row, over the live parts (lse != -inf):
//   L = max lse_j,  lse = L + ln sum exp(lse_j - L),  out = sum exp(lse_j - lse) o_j.
// A part with lse = -inf is skipped (its o is never read, so a NaN there
// cannot leak); no live part gives out = 0, lse = -inf.  The wave reads the
// row's part lse values lane-parallel (lane j holds part j), reduces max and
// sum across the wave, and then visits only the live parts, eight at a time,
// with each lane moving two 16-byte vectors per part (columns 4*lane and
// 256 + 4*lane), so that sixteen loads per lane are in flight instead of one
// part at a time.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mla_kernels.h"

namespace mla {
namespace rowmerge {

typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kBatch = 8;                    // parts in flight per wave

// Reductions over the 64 lanes of a wave, all in VGPRs: the gfx950 row-swap
// permutes pair lane l with l ^ 32 and then with l ^ 16 (with both operands
// holding v, the two results at a lane are v[l] and its partner's value);
// row rotations by 8, 4, 2 and 1 lanes (DPP) then cover the 16 lanes of a
// row.  Every lane ends with the same value: each step combines the same two
// values at both lanes of a pair, in either order.
template <typename Op>
__device__ __forceinline__ float wave_reduce(float v, Op op) {
  uint32_t u = __float_as_uint(v);
  const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  v = op(__uint_as_float(a[0]), __uint_as_float(a[1]));
  u = __float_as_uint(v);
  const auto b = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  v = op(__uint_as_float(b[0]), __uint_as_float(b[1]));
  // DPP row_ror:n = 0x120 + n
  v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xf, 0xf, false)));
  v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x124, 0xf, 0xf, false)));
  v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x122, 0xf, 0xf, false)));
  v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x121, 0xf, 0xf, false)));
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
  return wave_reduce(v, [](float x, float y) { return fmaxf(x, y); });
}

__device__ __forceinline__ float wave_sum(float v) {
  return wave_reduce(v, [](float x, float y) { return x + y; });
}

// A lane's value read by every lane (src wave-uniform).
__device__ __forceinline__ float lane_value(float v, int src) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), src));
}

// Part rows as fp32 (callers' partials) or as fp16 divided by a per-row
// scale (the split-K workspace): a lane loads columns 4 lane .. +3 and
// 256 + 4 lane .. +3 as raw values (load_raw) and converts them to fp32 where
// it uses them (cvt), so that the loads of several parts are in flight at once.
struct F32Rows {
  typedef f32x4_t Raw;
  template <typename RowAt>
  __device__ __forceinline__ static void load_raw(RowAt row_at, int j, int lane, Raw& v0, Raw& v1) {
    const float* r = row_at(j);
    v0 = *(const f32x4_t*)(r + 4 * lane);
    v1 = *(const f32x4_t*)(r + 256 + 4 * lane);
  }
  __device__ __forceinline__ static f32x4_t cvt(Raw v) { return v; }
};

typedef _Float16 f16x4_t __attribute__((ext_vector_type(4)));
typedef uint16_t u16x4_t __attribute__((ext_vector_type(4)));

// bf16 -> fp32 is exact: the bf16 bits are the upper half of the fp32 bits.
__device__ __forceinline__ f32x4_t bf16x4_f32(u16x4_t a) {
  return f32x4_t{__uint_as_float((uint32_t)a[0] << 16), __uint_as_float((uint32_t)a[1] << 16),
                 __uint_as_float((uint32_t)a[2] << 16), __uint_as_float((uint32_t)a[3] << 16)};
}

// Rows of wire-form parts: bf16.
struct Bf16Rows {
  typedef u16x4_t Raw;
  template <typename RowAt>
  __device__ __forceinline__ static void load_raw(RowAt row_at, int j, int lane, Raw& v0, Raw& v1) {
    const uint16_t* r = row_at(j);
    v0 = *(const u16x4_t*)(r + 4 * lane);
    v1 = *(const u16x4_t*)(r + 256 + 4 * lane);
  }
  __device__ __forceinline__ static f32x4_t cvt(Raw a) { return bf16x4_f32(a); }
};

struct F16Rows {
  typedef f16x4_t Raw;
  template <typename RowAt>
  __device__ __forceinline__ static void load_raw(RowAt row_at, int j, int lane, Raw& v0, Raw& v1) {
    const uint16_t* r = row_at(j);
    v0 = *(const f16x4_t*)(r + 4 * lane);
    v1 = *(const f16x4_t*)(r + 256 + 4 * lane);
  }
  __device__ __forceinline__ static f32x4_t cvt(Raw a) {
    return f32x4_t{(float)a[0], (float)a[1], (float)a[2], (float)a[3]};
  }
};

// Merge n parts of one row.  lse_at(j): part j's lse; row_at(j): part j's
// row (Rows says how to read it); scale_at(j): the factor part j's stored
// values carry (1 for fp32 parts).  Leaves the lane's outputs (columns
// 4 lane .. +3 and 256 + 4 lane .. +3) in acc0, acc1 and returns the merged
// lse.
template <typename Rows, typename LseAt, typename RowAt, typename ScaleAt>
__device__ __forceinline__ float merge_row(int n, LseAt lse_at, RowAt row_at, ScaleAt scale_at,
                                           f32x4_t& acc0, f32x4_t& acc1, int lane) {
  float m = -INFINITY;
  for (int j0 = 0; j0 < n; j0 += 64) {
    const int j = j0 + lane;
    if (j < n) m = fmaxf(m, lse_at(j));
  }
  m = wave_max(m);
  acc0 = f32x4_t{0.f, 0.f, 0.f, 0.f};
  acc1 = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float lse = -INFINITY;
  if (m != -INFINITY) {
    float s = 0.f;
    for (int j0 = 0; j0 < n; j0 += 64) {
      const int j = j0 + lane;
      const float l = j < n ? lse_at(j) : -INFINITY;
      if (l != -INFINITY) s += __expf(l - m);
    }
    lse = m + __logf(wave_sum(s));
    for (int j0 = 0; j0 < n; j0 += 64) {
      const int j = j0 + lane;
      const float l = j < n ? lse_at(j) : -INFINITY;
      const float w = l != -INFINITY ? __expf(l - lse) * scale_at(j) : 0.f;
      uint64_t live = __ballot(l != -INFINITY);
      while (live) {
        int idx[kBatch];
        int cnt = 0;
#pragma unroll
        for (int k = 0; k < kBatch; ++k) {
          idx[k] = live ? __builtin_ctzll(live) : idx[0];
          if (live) {
            live &= live - 1;
            ++cnt;
          }
        }
        // raw values first (converted at use), so that no load waits for another
        typename Rows::Raw v0[kBatch], v1[kBatch];
#pragma unroll
        for (int k = 0; k < kBatch; ++k)
          if (k < cnt) Rows::load_raw(row_at, j0 + idx[k], lane, v0[k], v1[k]);
#pragma unroll
        for (int k = 0; k < kBatch; ++k) {
          if (k < cnt) {
            const float wk = lane_value(w, idx[k]);
            acc0 += wk * Rows::cvt(v0[k]);
            acc1 += wk * Rows::cvt(v1[k]);
          }
        }
      }
    }
  }
  return lse;
}

// Stores of a merged row: fp32, or bf16 rounded to nearest even.
__device__ __forceinline__ void store_row(float* out, f32x4_t acc0, f32x4_t acc1, int lane) {
  *(f32x4_t*)(out + 4 * lane) = acc0;
  *(f32x4_t*)(out + 256 + 4 * lane) = acc1;
}

__device__ __forceinline__ u16x4_t f32x4_bf16(f32x4_t v) {
  return u16x4_t{__builtin_bit_cast(uint16_t, (__bf16)v[0]), __builtin_bit_cast(uint16_t, (__bf16)v[1]),
                 __builtin_bit_cast(uint16_t, (__bf16)v[2]), __builtin_bit_cast(uint16_t, (__bf16)v[3])};
}

__device__ __forceinline__ void store_row(uint16_t* out, f32x4_t acc0, f32x4_t acc1, int lane) {
  *(u16x4_t*)(out + 4 * lane) = f32x4_bf16(acc0);
  *(u16x4_t*)(out + 256 + 4 * lane) = f32x4_bf16(acc1);
}


// merge_row in one trip to memory: with n <= N parts, every part's row is
// requested together with its lse, instead of the lse first and then the live
// rows eight parts at a time.  The N loads are unconditional (parts past n
// re-read part n - 1, which the cache serves).  Rows of dead parts are read
// but never enter the sum: with kGuard (callers' parts, which may hold NaN
// there) a part is added only when live; without it (the split-K workspace,
// whose rows are always finite) a dead part is added with weight 0.  Same
// arithmetic and order as merge_row.  n >= 1 (the merge takes 1..64 parts,
// the combine two splits or more).
template <int N, bool kGuard, typename Rows, typename LseAt, typename RowAt, typename ScaleAt>
__device__ __forceinline__ float merge_row_one_trip(int n, LseAt lse_at, RowAt row_at,
                                                    ScaleAt scale_at, f32x4_t& acc0,
                                                    f32x4_t& acc1, int lane) {
  const float l = lane < n ? lse_at(lane) : -INFINITY;
  const float sc = lane < n ? scale_at(lane) : 0.f;
  // raw values first (converted at use), so that no load waits for another
  typename Rows::Raw v0[N], v1[N];
#pragma unroll
  for (int j = 0; j < N; ++j) Rows::load_raw(row_at, j < n ? j : n - 1, lane, v0[j], v1[j]);
  __builtin_amdgcn_sched_barrier(0);  // every load issued before the reductions
  acc0 = f32x4_t{0.f, 0.f, 0.f, 0.f};
  acc1 = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // no branch on an all-dead row (m = -inf): its weights are all 0 and its
  // lse comes out as ln 0 = -inf, and the loads stay ahead of the reductions
  float m = wave_max(l);
  m = m == -INFINITY ? 0.f : m;
  const float lse = m + __logf(wave_sum(l != -INFINITY ? __expf(l - m) : 0.f));
  const float w = l != -INFINITY ? __expf(l - lse) * sc : 0.f;
  const uint64_t live = __ballot(l != -INFINITY);
#pragma unroll
  for (int j = 0; j < N; ++j) {
    const float wj = lane_value(w, j);
    const f32x4_t a0 = acc0 + wj * Rows::cvt(v0[j]);
    const f32x4_t a1 = acc1 + wj * Rows::cvt(v1[j]);
    const bool take = !kGuard || ((live >> j) & 1);
    acc0 = take ? a0 : acc0;
    acc1 = take ? a1 : acc1;
  }
  return lse;
}

constexpr int kOneTrip = 16;

template <bool kGuard, typename Rows, typename LseAt, typename RowAt, typename ScaleAt>
__device__ __forceinline__ float merge_parts(int n, LseAt lse_at, RowAt row_at, ScaleAt scale_at,
                                             f32x4_t& acc0, f32x4_t& acc1, int lane) {
  if (n <= 4) return merge_row_one_trip<4, kGuard, Rows>(n, lse_at, row_at, scale_at, acc0, acc1, lane);
  if (n <= 8) return merge_row_one_trip<8, kGuard, Rows>(n, lse_at, row_at, scale_at, acc0, acc1, lane);
  if (n <= kOneTrip)
    return merge_row_one_trip<kOneTrip, kGuard, Rows>(n, lse_at, row_at, scale_at, acc0, acc1, lane);
  return merge_row<Rows>(n, lse_at, row_at, scale_at, acc0, acc1, lane);
}

// Split-K combine of one row (r, row) of a job's S split rows in the
// workspace (split j at index (r S + j) rows + row): the merged row and lse
// to the caller's output, or in the wire form the bf16 row and (m, l).  P is
// any parameter block with the workspace and output fields of CombineParams.
template <typename P>
__device__ __forceinline__ void combine_row(const P& p, int S, int r, int row, int lane) {
  const int64_t base = (int64_t)r * S * p.rows + row;  // split j of (r, row) at base + j*rows
  const int i = row / p.H, h = row - (row / p.H) * p.H;
  const int64_t oo = r * p.out_s0 + i * p.out_s1 + h * p.out_s2;
  auto lse_at = [&](int j) { return p.ws_lse[base + (int64_t)j * p.rows]; };
  auto row16 = [&](int j) { return p.ws_o16 + (base + (int64_t)j * p.rows) * kDLat; };
  auto row32 = [&](int j) { return p.ws_o32 + (base + (int64_t)j * p.rows) * kDLat; };
  auto scale16 = [&](int j) { return p.ws_scale[base + (int64_t)j * p.rows]; };
  auto one = [](int) { return 1.f; };
  f32x4_t acc0, acc1;
  float lse;
  lse = p.ws_f16 ? merge_parts<false, F16Rows>(S, lse_at, row16, scale16, acc0, acc1, lane)
                 : merge_parts<false, F32Rows>(S, lse_at, row32, one, acc0, acc1, lane);
  const int64_t lo = r * p.lse_s0 + i * p.lse_s1 + h * p.lse_s2;
  if (!p.out_wire) {
    store_row(p.out + oo, acc0, acc1, lane);
    if (lane == 0) p.lse[lo] = lse;
    return;
  }
  // wire form: bf16 row, and (m, l) with m the largest score over the splits
  // (their maxima, log2 units) and l = exp(lse - m)
  store_row(p.out16 + oo, acc0, acc1, lane);
  float m2 = -INFINITY;
  for (int j0 = 0; j0 < S; j0 += 64) {
    const int j = j0 + lane;
    if (j < S) m2 = fmaxf(m2, p.ws_max[base + (int64_t)j * p.rows]);
  }
  m2 = wave_max(m2);
  if (lane == 0) {
    const float m = m2 * 0.69314718055994530942f;
    p.lse[lo] = lse == -INFINITY ? -INFINITY : m;
    p.lse[lo + 1] = lse == -INFINITY ? 0.f : __expf(lse - m);
  }
}

}  // namespace rowmerge
}  // namespace mla
