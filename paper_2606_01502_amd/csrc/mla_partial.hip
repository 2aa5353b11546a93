// Sparse absorbed-MLA partial attention for gfx950 (MI355X).
//
// One workgroup (NW = 8 or 4 waves) handles one (job, row tile of 16*NW
// rows, slot range).  The rows
// of a job (Mq x H query rows; a row is a 512-wide latent part plus a 64-wide
// decoupled-RoPE part, the paper's d_qk = 576 wire row of Section 3.2) share
// one selection of 64-token cache blocks, so each selected block is read from
// HBM once per workgroup and staged in LDS for all rows:
//
//   gather   direct-to-LDS 16-byte loads (global_load_lds_dwordx4) of each
//            selected block, 32 tokens (36 KiB) at a time, into a ring of four
//            LDS buffers; up to three half-blocks are in flight while one is
//            computed.  The chunk's block table maps the selected logical
//            block to its pool block.
//   S^T      = K . Q^T per wave for its 16 rows: bf16 MFMA 16x16x32, K read
//            from LDS (b128), Q held in registers for the whole kernel.
//   softmax  online, in the exp2 domain, with wavefront reductions; the
//            running max is only moved when a block raises it by more than
//            2^8, so the accumulator is rarely rescaled (exact either way).
//   P        bf16 probabilities go through a small swizzled LDS tile so every
//            wave sees all rows.
//   O^T     += V^T . P^T per wave for its 512/NW latent columns and all rows
//            of the tile: bf16 MFMA, V^T read with the transposing LDS read
//            (ds_read_b64_tr_b16) from the same staged tile, since the value
//            is the latent part of the key (Section 3.2).
//   epilogue normalised output and lse = max + ln(sum) per row, either to the
//            caller's buffers or, under split-K, to a workspace that the
//            combine kernel reduces with the merge algebra (Section 3.3).
//
// LDS swizzles (token t within a half-block, 16-byte chunk c within a row):
//   latent rows (1 KiB):   chunk c lives in slot c ^ ((t & 15) ^ ((t & 16) >> 2))
//   RoPE rows (128 B):     chunk c lives in slot c ^ ((t >> 1) & 7)
//   P rows (64 B):         chunk c lives in slot c ^ ((row >> 2) & 3)
// so the b128 key reads, the transposing value reads and the P reads all hit
// distinct banks at the minimum number of LDS cycles.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mla_kernels.h"

namespace mla {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef int i32x2_t __attribute__((ext_vector_type(2)));
typedef int i32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

#define LDS __attribute__((address_space(3)))
#define GLOBAL __attribute__((address_space(1)))

constexpr int kNumBuf = 4;
constexpr int kHalfTokens = 32;
constexpr int kHalfCkvBytes = kHalfTokens * kDLat * 2;  // 32 KiB
constexpr int kHalfKpeBytes = kHalfTokens * kDPe * 2;   // 4 KiB
constexpr int kHalfBytes = kHalfCkvBytes + kHalfKpeBytes;
constexpr int kLoadsPerHalf = 9;  // per wave: 8 latent rows + 1 KiB of RoPE rows
constexpr float kTau = 8.0f;      // lazy-rescale threshold, log2 units
constexpr float kLn2 = 0.69314718055994530942f;

// s_waitcnt immediate (gfx9 encoding) that waits for vmcnt <= n only.
constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

template <int NW>
struct Lds {
  static constexpr int kRowsWg = 16 * NW;
  static constexpr int kP = kNumBuf * kHalfBytes;
  static constexpr int kAlpha = kP + kRowsWg * kHalfTokens * 2;
  static constexpr int kEll = kAlpha + kRowsWg * 4;
  static constexpr int kFlags = kEll + kRowsWg * 4;
  static constexpr int kWaveCnt = kFlags + 4 * NW;
  static constexpr int kList = kWaveCnt + 4 * NW;
  static constexpr int kTotal = kList + kMaxSlotsPerSplit * 4;
};
static_assert(Lds<8>::kTotal <= 160 * 1024, "LDS budget");

__device__ __forceinline__ void dma16(const uint8_t* src, LDS uint8_t* dst) {
  __builtin_amdgcn_global_load_lds((const GLOBAL void*)src, (LDS void*)dst, 16, 0, 0);
}

__device__ __forceinline__ bf16x8_t lds_b128(const LDS uint8_t* p) {
  return *(const LDS bf16x8_t*)p;
}

// Four transposing LDS reads (ds_read_b64_tr_b16) issued back to back, then
// one wait for all of them.  Written as one asm block because the compiler
// treats the builtin form as possibly reading the buffers that outstanding
// direct-to-LDS prefetches write and would wait for all of them (vmcnt(0))
// first; here those buffers are known to be disjoint from the one read.
// The results are declared as pairs of 32-bit lanes: a 4 x 16-bit asm output
// is not carried through whole by the compiler.
__device__ __forceinline__ void lds_tr16_x4(i32x2_t& r0, i32x2_t& r1, i32x2_t& r2, i32x2_t& r3,
                                            const LDS uint8_t* base, int o0, int o1, int o2,
                                            int o3) {
  const uint32_t b = (uint32_t)(uintptr_t)base;
  asm volatile(
      "ds_read_b64_tr_b16 %0, %4\n\t"
      "ds_read_b64_tr_b16 %1, %5\n\t"
      "ds_read_b64_tr_b16 %2, %6\n\t"
      "ds_read_b64_tr_b16 %3, %7\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(r0), "=&v"(r1), "=&v"(r2), "=&v"(r3)
      : "v"(b + o0), "v"(b + o1), "v"(b + o2), "v"(b + o3)
      : "memory");
}

__device__ __forceinline__ f32x4_t mfma(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float xor_max(float v) {
  v = fmaxf(v, __shfl_xor(v, 16));
  return fmaxf(v, __shfl_xor(v, 32));
}

__device__ __forceinline__ float xor_sum(float v) {
  v += __shfl_xor(v, 16);
  return v + __shfl_xor(v, 32);
}

// Workgroup barrier for LDS traffic only.  __syncthreads() would also wait
// for every outstanding vector-memory operation, including the direct-to-LDS
// prefetches of later half-blocks; here each wave waits for its own LDS
// reads/writes, and the prefetches are waited for explicitly by vmcnt.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Direct-to-LDS loads a wave issues per half-block (latent rows + RoPE rows).
template <int NW>
__device__ __forceinline__ int loads_per_half(int wave) {
  return kHalfTokens / NW + (wave < 4 ? 1 : 0);
}

// Issue the direct-to-LDS loads of half-block `half` of pool block b:
// wave w loads latent rows w*(32/NW) .. +32/NW-1 (1 KiB each, chunks
// permuted by the row's swizzle) and, for w < 4, RoPE rows 8w .. 8w+7.
template <int NW>
__device__ __forceinline__ void issue_half(const PartialParams& p, int64_t b, int half,
                                           LDS uint8_t* buf, int wave, int lane_in) {
  constexpr int kRowsPerWave = kHalfTokens / NW;
  // Recompute the per-lane source offsets at every issue instead of letting
  // them be hoisted out of the main loop: registers are the scarce resource
  // there, and a spill would make the scratch reload wait for every
  // outstanding prefetch.
  int lane;
  asm volatile("v_mov_b32 %0, %1" : "=v"(lane) : "v"(lane_in));
  const uint8_t* ckv = p.ckv + (b * kBlock + half * kHalfTokens) * (kDLat * 2);
#pragma unroll
  for (int j = 0; j < kRowsPerWave; ++j) {
    const int t = wave * kRowsPerWave + j;
    const int f = (t & 15) ^ ((t & 16) >> 2);
    dma16(ckv + t * (kDLat * 2) + ((lane ^ f) << 4), buf + t * (kDLat * 2));
  }
  if (wave < 4) {
    const uint8_t* kpe = p.kpe + (b * kBlock + half * kHalfTokens) * (kDPe * 2);
    const int t = wave * 8 + (lane >> 3);
    const int c = (lane & 7) ^ ((t >> 1) & 7);
    dma16(kpe + t * (kDPe * 2) + (c << 4), buf + kHalfCkvBytes + wave * 1024);
  }
}

__device__ __forceinline__ void wait_vm(int n) {
  // vmcnt is a 6-bit counter; n <= 2 * 9 here
  switch (n) {
    case 0: __builtin_amdgcn_s_waitcnt(waitcnt_vm(0)); break;
    case 4: __builtin_amdgcn_s_waitcnt(waitcnt_vm(4)); break;
    case 5: __builtin_amdgcn_s_waitcnt(waitcnt_vm(5)); break;
    case 8: __builtin_amdgcn_s_waitcnt(waitcnt_vm(8)); break;
    case 9: __builtin_amdgcn_s_waitcnt(waitcnt_vm(9)); break;
    case 10: __builtin_amdgcn_s_waitcnt(waitcnt_vm(10)); break;
    case 16: __builtin_amdgcn_s_waitcnt(waitcnt_vm(16)); break;
    case 18: __builtin_amdgcn_s_waitcnt(waitcnt_vm(18)); break;
    default: __builtin_amdgcn_s_waitcnt(waitcnt_vm(0)); break;
  }
}

// NW waves: wave w computes S^T and the softmax for rows 16w .. 16w+15 of the
// row tile, and O^T for latent columns w*512/NW .. (w+1)*512/NW - 1 of every
// row of the tile.
template <int NW>
__global__ __launch_bounds__(NW * 64) void partial_bf16_kernel(const PartialParams p) {
  using L = Lds<NW>;
  constexpr int kRowsWg = L::kRowsWg;
  constexpr int kDT = kDLat / NW / 16;  // 16-column tiles per wave
  __shared__ __attribute__((aligned(16))) uint8_t smem_raw[L::kTotal];
  LDS uint8_t* smem = (LDS uint8_t*)smem_raw;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n16 = lane & 15;  // MFMA column / row-in-group index
  const int g = lane >> 4;    // MFMA k-group

  // ---- work item
  const int w_id = blockIdx.x;
  const int s_idx = w_id % p.n_splits;
  const int rt = (w_id / p.n_splits) % p.row_tiles;
  const int r = w_id / (p.n_splits * p.row_tiles);
  const int slot0 = s_idx * p.slots_per_split;
  const int nslots = max(0, min(p.K - slot0, p.slots_per_split));

  // ---- compact the valid selected blocks of the slot range (slot order kept)
  LDS int* list = (LDS int*)(smem + L::kList);
  LDS int* wave_cnt = (LDS int*)(smem + L::kWaveCnt);
  int n_valid = 0;
  for (int base = 0; base < nslots; base += NW * 64) {
    const int i = base + tid;
    int b = -1;
    if (i < nslots) {
      const int id = p.sel[r * p.sel_s0 + slot0 + i];
      if (id >= 0 && id < p.NB) {
        const int bb = p.table[r * p.table_s0 + id];
        if (bb >= 0 && bb < p.P) b = bb;
      }
    }
    const uint64_t m = __ballot(b >= 0);
    const int before = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) wave_cnt[wave] = __popcll(m);
    __syncthreads();
    int off = n_valid, total = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const int c = wave_cnt[w];
      off += (w < wave) ? c : 0;
      total += c;
    }
    if (b >= 0) list[off + before] = b;
    n_valid += total;
    __syncthreads();
  }

  // ---- this wave's 16 query rows as MFMA B operands, held for the whole kernel
  const int row_wg0 = rt * kRowsWg;
  const int own_row_l = wave * 16 + n16;  // row within the tile owned by this lane
  bf16x8_t qb[18];
  {
    const int row = row_wg0 + own_row_l;
    if (row < p.rows) {
      const int i = row / p.H, h = row - (row / p.H) * p.H;
      const uint16_t* ql = p.q_lat + r * p.ql_s0 + i * p.ql_s1 + h * p.ql_s2 + g * 8;
      const uint16_t* qp = p.q_pe + r * p.qp_s0 + i * p.qp_s1 + h * p.qp_s2 + g * 8;
#pragma unroll
      for (int ks = 0; ks < 16; ++ks) qb[ks] = *(const bf16x8_t*)(ql + ks * 32);
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) qb[16 + ks] = *(const bf16x8_t*)(qp + ks * 32);
    } else {
#pragma unroll
      for (int ks = 0; ks < 18; ++ks) qb[ks] = bf16x8_t{};
    }
  }
  // Q is resident before the first prefetch is issued, so that the only
  // vector-memory operations in flight inside the main loop are prefetches.
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));

  f32x4_t O[kDT][NW];
#pragma unroll
  for (int dt = 0; dt < kDT; ++dt)
#pragma unroll
    for (int rg = 0; rg < NW; ++rg) O[dt][rg] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  LDS float* alpha_lds = (LDS float*)(smem + L::kAlpha);
  LDS int* flags = (LDS int*)(smem + L::kFlags);
  const int my_loads = loads_per_half<NW>(wave);

  // ---- main loop over half-blocks
  const int n_half = 2 * n_valid;
  for (int h = 0; h < n_half && h < 3; ++h)
    issue_half<NW>(p, list[h >> 1], h & 1, smem + (h % kNumBuf) * kHalfBytes, wave, lane);

  for (int h = 0; h < n_half; ++h) {
    wait_vm(min(n_half - 1 - h, 2) * my_loads);
    lds_barrier();  // half h is in LDS; every wave is done with half h-1
    if (h + 3 < n_half)
      issue_half<NW>(p, list[(h + 3) >> 1], (h + 3) & 1, smem + ((h + 3) % kNumBuf) * kHalfBytes,
                     wave, lane);
    const LDS uint8_t* cb = smem + (h % kNumBuf) * kHalfBytes;

    // Per-lane LDS offsets are recomputed from an opaque copy of the lane id in
    // every iteration (a few VALU ops) rather than held in registers across
    // the loop, which would push the kernel past 256 VGPRs.
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int ln16 = ln & 15, lg = ln >> 4;

    // S^T[token][row] for this wave's rows, tokens 16*tau + (0..15).
    // Key chunk 4ks+g of token 16*tau+ln16 sits in slot (4ks+g) ^ ln16 ^ 4tau,
    // i.e. at key_base ^ ((((ks & 3) ^ tau)) << 6) + (ks >> 2) * 256.
    const int key_base = ln16 * 1024 + ((lg ^ (ln16 & 3)) << 4) + ((ln16 >> 2) << 6);
    const int rope_base = kHalfCkvBytes + ln16 * 128;
    f32x4_t acc[2] = {f32x4_t{0.f, 0.f, 0.f, 0.f}, f32x4_t{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int tau = 0; tau < 2; ++tau)
        acc[tau] = mfma(lds_b128(cb + tau * 2048 + rope_base + (((4 * kk + lg) ^ (ln16 >> 1)) << 4)),
                        qb[16 + kk], acc[tau]);
#pragma unroll
    for (int ks = 0; ks < 16; ++ks)
#pragma unroll
      for (int tau = 0; tau < 2; ++tau)
        acc[tau] = mfma(lds_b128(cb + tau * 16384 + (ks >> 2) * 256 + (key_base ^ ((((ks & 3) ^ tau)) << 6))),
                        qb[ks], acc[tau]);

    // online softmax over the half's 32 tokens, own rows (exp2 domain)
    float tv[8];
    float bm = -INFINITY;
#pragma unroll
    for (int tau = 0; tau < 2; ++tau)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        tv[tau * 4 + i] = acc[tau][i] * p.scale_log2;
        bm = fmaxf(bm, tv[tau * 4 + i]);
      }
    bm = xor_max(bm);
    float alpha = 1.f;
    int rescaled = 0;
    if (bm > m_run + kTau) {
      if (m_run != -INFINITY) {
        alpha = __builtin_amdgcn_exp2f(m_run - bm);
        rescaled = 1;
      }
      l_run *= alpha;
      m_run = bm;
    }
    if (g == 0) alpha_lds[own_row_l] = alpha;
    float ps = 0.f;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      tv[k] = __builtin_amdgcn_exp2f(tv[k] - m_run);
      ps += tv[k];
    }
    l_run += ps;
#pragma unroll
    for (int tau = 0; tau < 2; ++tau) {
      bf16x4_t pk;
#pragma unroll
      for (int i = 0; i < 4; ++i) pk[i] = (__bf16)tv[tau * 4 + i];
      const int c = 2 * tau + (g >> 1);
      *(LDS bf16x4_t*)(smem + L::kP + own_row_l * 64 + ((c ^ ((own_row_l >> 2) & 3)) << 4) +
                       ((g & 1) << 3)) = pk;
    }
    const int wave_rescaled = __ballot(rescaled) != 0;
    if (lane == 0) flags[wave] = wave_rescaled;
    lds_barrier();  // P, alpha and flags of every row are in LDS

    int any_flag = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) any_flag |= flags[w];
    if (any_flag) {
#pragma unroll
      for (int rg = 0; rg < NW; ++rg) {
        const float a = alpha_lds[16 * rg + n16];
#pragma unroll
        for (int dt = 0; dt < kDT; ++dt) O[dt][rg] *= a;
      }
    }
    // Transposing value reads: lane (g, r4 = (lane>>2)&3, q4 = lane&3) supplies
    // token 8g + 4hh + r4 and latent columns 16*ct + 4*q4 .. +3; the result
    // gives lane n16 column 16*ct + n16 of four consecutive tokens.
    int lv = lane;
    asm volatile("" : "+v"(lv));
    const int r4 = (lv >> 2) & 3, q4 = lv & 3, vg = lv >> 4;
    int tr_off[2];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int t = 8 * vg + 4 * hh + r4;
      const int f = (t & 15) ^ ((t & 16) >> 2);
      const int c0 = 2 * wave * kDT + (q4 >> 1);  // chunk of column tile ct = wave*kDT
      // chunk 2*dt + c0 of token t sits in slot (c0 + 2dt) ^ f; the 2dt bits
      // are disjoint from c0's, so the slot is ((c0 ^ f) ^ 2dt) within the
      // 16-chunk group of c0
      tr_off[hh] = t * 1024 + ((q4 & 1) << 3) + (((c0 & ~15) | ((c0 & 15) ^ f)) << 4);
    }
    bf16x8_t va[kDT];
#pragma unroll
    for (int dt = 0; dt < kDT; dt += 2) {
      i32x2_t lo0, hi0, lo1, hi1;
      lds_tr16_x4(lo0, hi0, lo1, hi1, cb, tr_off[0] ^ (dt << 5), tr_off[1] ^ (dt << 5),
                  tr_off[0] ^ ((dt + 1) << 5), tr_off[1] ^ ((dt + 1) << 5));
      va[dt] = __builtin_bit_cast(bf16x8_t, i32x4_t{lo0[0], lo0[1], hi0[0], hi0[1]});
      va[dt + 1] = __builtin_bit_cast(bf16x8_t, i32x4_t{lo1[0], lo1[1], hi1[0], hi1[1]});
    }
    // P tile (rows x 32 tokens, bf16, 64 B per row): row 16*rg + n16 of the
    // tile at p_rd + rg * 1024 (its swizzle only depends on n16)
    const int p_rd = L::kP + (lv & 15) * 64 + ((vg ^ (((lv & 15) >> 2) & 3)) << 4);
#pragma unroll
    for (int rg = 0; rg < NW; ++rg) {
      const bf16x8_t pb = lds_b128(smem + p_rd + rg * 1024);
#pragma unroll
      for (int dt = 0; dt < kDT; ++dt) O[dt][rg] = mfma(va[dt], pb, O[dt][rg]);
    }
  }

  // ---- epilogue: row statistics of own rows, then every wave normalises its columns
  LDS float* ell_lds = (LDS float*)(smem + L::kEll);
  const bool direct = p.n_splits == 1;
  const int64_t part = (int64_t)r * p.n_splits + s_idx;
  {
    const float l_tot = xor_sum(l_run);
    const int row = row_wg0 + own_row_l;
    if (g == 0) {
      ell_lds[own_row_l] = l_tot;
      if (row < p.rows) {
        const float lse = l_tot > 0.f ? (m_run + __log2f(l_tot)) * kLn2 : -INFINITY;
        if (direct) {
          const int i = row / p.H, hd = row - (row / p.H) * p.H;
          p.lse[r * p.lse_s0 + i * p.lse_s1 + hd * p.lse_s2] = lse;
        } else {
          p.ws_lse[part * p.rows + row] = lse;
        }
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int rg = 0; rg < NW; ++rg) {
    const int row = row_wg0 + 16 * rg + n16;
    if (row >= p.rows) continue;
    const float l_tot = ell_lds[16 * rg + n16];
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    float* dst;
    if (direct) {
      const int i = row / p.H, hd = row - (row / p.H) * p.H;
      dst = p.out + r * p.out_s0 + i * p.out_s1 + hd * p.out_s2;
    } else {
      dst = p.ws_o + (part * p.rows + row) * kDLat;
    }
    dst += wave * (kDT * 16) + 4 * g;
#pragma unroll
    for (int dt = 0; dt < kDT; ++dt) *(f32x4_t*)(dst + dt * 16) = O[dt][rg] * inv;
  }
}

}  // namespace

hipError_t launch_partial(const PartialParams& p, int R, bool fp8, int waves, hipStream_t s) {
  if (fp8) return hipErrorNotSupported;
  const int grid = R * p.row_tiles * p.n_splits;
  if (grid <= 0) return hipSuccess;
  if (waves == 8)
    hipLaunchKernelGGL(partial_bf16_kernel<8>, dim3(grid), dim3(8 * 64), 0, s, p);
  else
    hipLaunchKernelGGL(partial_bf16_kernel<4>, dim3(grid), dim3(4 * 64), 0, s, p);
  return hipGetLastError();
}

}  // namespace mla
