// Sparse absorbed-MLA partial attention for gfx950 (MI355X).
//
// One workgroup of 4 waves handles one (job, row tile, slot range).  The rows
// of a job (Mq x H query rows; a row is a 512-wide latent part plus a 64-wide
// decoupled-RoPE part, the paper's d_qk = 576 wire row of Section 3.2) share
// one selection of 64-token cache blocks, so each selected block is read from
// HBM once per workgroup and staged in LDS for all of its rows:
//
//   gather   direct-to-LDS 16-byte loads (global_load_lds_dwordx4) of each
//            selected block into LDS, one block (bf16, 72 KiB) or three (fp8
//            e4m3 codes, 36 KiB) ahead of the block being computed.  The
//            chunk's block table maps the selected logical block to its pool
//            block.  Blocks land swizzled, in the layout the reads below use.
//   S^T      = K . Q^T per wave for its 16*RG rows: bf16 MFMA 16x16x32, K read
//            from LDS (16-byte reads of bf16, or 8-byte reads of e4m3 codes
//            converted to bf16 in registers, exactly, between the products),
//            Q held in registers for the whole kernel.
//   softmax  online, in the exp2 domain, with wavefront reductions; the
//            running max only moves when a block raises it by more than 2^8,
//            so the accumulator is rarely rescaled (exact either way).
//   O^T     += V^T . P^T per wave for its rows and all 512 latent columns:
//            bf16 MFMA with P^T taken straight from the S^T accumulator layout
//            (the k index of the product is a fixed permutation of the block's
//            tokens) and V^T read with the transposing LDS read
//            (ds_read_b64_tr_b16, or ds_read_b64_tr_b8 and a conversion in
//            registers for fp8) from the same stage, since the value is the
//            latent part of the key (Section 3.2).  O lives in the
//            accumulation registers for the whole kernel.
//   epilogue normalised output and lse = max + ln(sum) per row, either to the
//            caller's buffers or, under split-K, to a workspace that the
//            combine kernel reduces with the merge algebra (Section 3.3).
//
// fp8 per-block scales (Section 6.3 mentions an FP8 sparse kernel; the scale
// granularity is this library's) stay out of the bf16 operands, which hold the
// codes exactly: the scores are multiplied by the block's scale and P by the
// same scale before its bf16 rounding.  With separate latent and RoPE scales
// (the kKvFp8Split instance) the RoPE part of the scores is first weighted by
// the RoPE / latent scale ratio, before the latent part is added.
//
// Selections (the SEL template parameter): one list of 64-token blocks per
// job (shared by its rows); one list per query row (a holder serving several
// routed requesters, Section 6.3), where a row tile loads the union of its
// rows' blocks once and masks every row to its own multiset; or single
// tokens (an indexer's top-k, Section 6.3's selection budgets), gathered 64
// at a time into the same stage layout, each with its own block's fp8
// scales.  Splits of a workspace of a megabyte or more store their rows as
// fp16 scaled by the row's largest magnitude.
//
// LDS swizzles (token t of the block, 16-byte chunk c of its row) are
// described with bf16_key and fp8_key below.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "mla_kernels.h"

namespace mla {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef short i16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef int i32x2_t __attribute__((ext_vector_type(2)));
typedef uint16_t u16x4_t __attribute__((ext_vector_type(4)));

#define LDS __attribute__((address_space(3)))
#define GLOBAL __attribute__((address_space(1)))

// LDS layout.  bf16 caches: two stages of one block each (64 latent rows of
// 1 KiB, then 64 RoPE rows of 128 B, swizzled as described at bf16_key);
// block h+1 streams in while block h is computed.  fp8 caches: four stages of
// one block of e4m3 codes each (64 latent rows of 512 B, then 64 RoPE rows of
// 64 B, swizzled as described at fp8_key); blocks h+1 .. h+3 stream in while
// block h is computed.  After the stages: the compacted pool-block list of
// the slot range and, for fp8, three floats per listed block (see
// fp8_factors).  The compactions' per-wave counters use the last bytes of the
// stage area, which no load writes before the compaction is over.
template <bool FP8>
struct Layout {
  static constexpr int kElt = FP8 ? 1 : 2;                     // bytes per element
  static constexpr int kRow = kDLat * kElt;                    // latent row
  static constexpr int kRopeRow = kDPe * kElt;                 // RoPE row
  static constexpr int kStage = kBlock * (kRow + kRopeRow);    // 72 KiB or 36 KiB
  static constexpr int kStageCkv = kBlock * kRow;
  static constexpr int kNum = FP8 ? 4 : 2;
  static constexpr int kLead = kNum - 1;  // blocks streaming ahead of the computed one
  static constexpr int kLoads = kStage / 1024 / 4;  // 1 KiB loads per wave per stage
  static constexpr int kList = kNum * kStage;
  static constexpr int kScales = kList + kMaxSlotsPerSplit * 4;
  static constexpr int kTotal = kScales + (FP8 ? kMaxSlotsPerSplit * 12 : 0);
  static constexpr int kWaveCnt = kNum * kStage - 16;
  // Per-row selections: a 64-bit row mask per list entry.  bf16: after the
  // rest, for a full list.  fp8 (whose four stages leave no room for that):
  // half a list, its scales and masks sharing the scale area.
  static constexpr int kPerRowCap = FP8 ? kMaxSlotsPerSplit / 2 : kMaxSlotsPerSplit;
  static constexpr int kMasks = FP8 ? kScales + kPerRowCap * 12 : kTotal;
  static constexpr int kTotalPerRow = FP8 ? kTotal : kMasks + kPerRowCap * 8;
};
static_assert(Layout<true>::kMasks + Layout<true>::kPerRowCap * 8 <= Layout<true>::kTotal,
              "fp8 per-row scales and masks fit the scale area");
static_assert(Layout<true>::kPerRowCap == kPerRowListFp8, "per-row fp8 list size");
static_assert(Layout<true>::kTotal <= 160 * 1024 && Layout<false>::kTotalPerRow <= 160 * 1024,
              "LDS budget");
static_assert(kPerRowCounterBytes <= Layout<false>::kWaveCnt && kPerRowCounterBytes <= Layout<true>::kWaveCnt,
              "per-row counters live in the stage area, below the wave counters");
constexpr float kTau = 8.0f;        // lazy-rescale threshold, log2 units
constexpr float kLn2 = 0.69314718055994530942f;

// s_waitcnt immediate (gfx9 encoding) that waits for vmcnt <= n only.
constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// One direct-to-LDS load per lane: 16 bytes from src to dst + 16 * lane (dst
// must be wave-uniform; it goes through M0).  Written as asm so that the
// compiler does not know about the LDS writes still in flight: otherwise it
// waits for them (vmcnt(0)) before every LDS read it cannot prove disjoint,
// including reads of the other buffer.  The code waits for the loads
// explicitly (vmcnt) before the barrier that publishes a buffer.
__device__ __forceinline__ void dma16(const uint8_t* src, LDS uint8_t* dst) {
  const uint32_t d = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)dst);
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(src), "s"(d) : "memory", "m0");
}

// The same with a wave-uniform 64-bit base in SGPRs and a 32-bit per-lane
// byte offset: the address needs no per-lane 64-bit arithmetic.
__device__ __forceinline__ void dma16s(const uint8_t* base, uint32_t off, LDS uint8_t* dst) {
  const uint32_t d = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)dst);
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(off), "s"(base), "s"(d) : "memory", "m0");
}

__device__ __forceinline__ bf16x8_t lds_b128(const LDS uint8_t* p) {
  return *(const LDS bf16x8_t*)p;
}

__device__ __forceinline__ f32x4_t mfma(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// S^T products with the accumulators in architectural VGPRs.  The compiler
// selects the accumulation-register form for every MFMA of a kernel that uses
// accumulation registers at all, and the 256 of them hold O here; these
// products are therefore written as inline asm with "v" operands.  Neither
// direction is interlocked: VALU code may read a product's result only 24
// wait states (a 16-pass XDL op) after it, and a product may read an operand
// that VALU code wrote only 3 wait states later.  The build checks the
// generated code for both (hazards.py).
// One S^T product, c += a . q (kFirst: c = a . q), as an asm statement of its
// own.  A wave issues in order and waits at a product until the matrix core
// takes it, so only what is placed between single products (key reads,
// loads of the next block) issues while the matrix core works; after a
// group of products it would overlap the group's last one only.  kPad ends
// with the 24 wait states after which VALU code may read c.
template <bool kFirst, bool kPad, bool kPre = false>
__device__ __forceinline__ void st1(f32x4_t& c, bf16x8_t a, bf16x8_t q) {
  // kPre: 3 wait states first, for operands just written by VALU code
  if constexpr (kFirst && kPre)
    asm volatile("s_nop 2\n\tv_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=&v"(c) : "v"(a), "v"(q));
  else if constexpr (kFirst)
    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=&v"(c) : "v"(a), "v"(q));
  else if constexpr (kPad && kPre)
    asm volatile("s_nop 2\n\tv_mfma_f32_16x16x32_bf16 %0, %1, %2, %0\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7"
                 : "+v"(c) : "v"(a), "v"(q));
  else if constexpr (kPad)
    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7"
                 : "+v"(c) : "v"(a), "v"(q));
  else if constexpr (kPre)
    asm volatile("s_nop 2\n\tv_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "v"(q));
  else
    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "v"(q));
}

// Ties the computation of x to this point of the instruction stream (an empty
// volatile asm that reads and writes x), so that the compiler cannot sink it
// down to its first use, next to the product that reads it.
template <typename T>
__device__ __forceinline__ void pin(T& x) {
  asm volatile("" : "+v"(x));
}

// x * s for an accumulator tile that lives in the accumulation registers.
// The empty asm statements keep the tile there: without them the register
// allocator moves part of O into architectural VGPRs for the whole kernel to
// serve these rare VALU uses, and spills.
__device__ __forceinline__ f32x4_t scale_acc(f32x4_t x, float s) {
  asm volatile("" : "+a"(x));
  x *= s;
  asm volatile("" : "+a"(x));
  return x;
}

// x *= s in the registers x already occupies.
__device__ __forceinline__ void scale_inplace(f32x4_t& x, float s) {
  float x0 = x[0], x1 = x[1], x2 = x[2], x3 = x[3];
  asm volatile("v_mul_f32 %0, %0, %4\n\tv_mul_f32 %1, %1, %4\n\tv_mul_f32 %2, %2, %4\n\t"
               "v_mul_f32 %3, %3, %4"
               : "+v"(x0), "+v"(x1), "+v"(x2), "+v"(x3)
               : "v"(s));
  x = f32x4_t{x0, x1, x2, x3};
}

// x[i] *= s[i] in the registers x already occupies.
__device__ __forceinline__ void scale_inplace4(f32x4_t& x, f32x4_t s) {
  float x0 = x[0], x1 = x[1], x2 = x[2], x3 = x[3];
  asm volatile("v_mul_f32 %0, %0, %4\n\tv_mul_f32 %1, %1, %5\n\tv_mul_f32 %2, %2, %6\n\t"
               "v_mul_f32 %3, %3, %7"
               : "+v"(x0), "+v"(x1), "+v"(x2), "+v"(x3)
               : "v"(s[0]), "v"(s[1]), "v"(s[2]), "v"(s[3]));
  x = f32x4_t{x0, x1, x2, x3};
}

// Four floats -> four bf16 (round to nearest even).
__device__ __forceinline__ u16x4_t f32x4_bf16(f32x4_t v) {
  return u16x4_t{__builtin_bit_cast(uint16_t, (__bf16)v[0]), __builtin_bit_cast(uint16_t, (__bf16)v[1]),
                 __builtin_bit_cast(uint16_t, (__bf16)v[2]), __builtin_bit_cast(uint16_t, (__bf16)v[3])};
}

// Two floats -> two fp16 (round to nearest even), packed low first.
__device__ __forceinline__ uint32_t pack_f16(float lo, float hi) {
  const _Float16 a = (_Float16)lo, b = (_Float16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

// Reductions over the four 16-lane rows of a wave (lanes l, l ^ 16, l ^ 32,
// l ^ 48) with the gfx950 row-swap permutes, which move data between VGPRs
// without a trip through LDS.  With both operands holding v, the 16-lane swap
// leaves {v[l], v[l ^ 16]} in the two results at every lane, and the 32-lane
// swap {v[l], v[l ^ 32]}.
__device__ __forceinline__ float xor_max(float v) {
  const uint32_t u = __float_as_uint(v);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const uint32_t w = __float_as_uint(v);
  const auto b = __builtin_amdgcn_permlane32_swap(w, w, false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ float xor_sum(float v) {
  const uint32_t u = __float_as_uint(v);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const uint32_t w = __float_as_uint(v);
  const auto b = __builtin_amdgcn_permlane32_swap(w, w, false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Workgroup barrier for LDS traffic only.  __syncthreads() would also wait
// for every outstanding vector-memory operation, including the direct-to-LDS
// prefetch of the next block; here each wave waits for its own LDS
// reads/writes, and the prefetch is waited for explicitly by vmcnt.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ __forceinline__ i16x4_t lds_tr16(const LDS uint8_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS i16x4_t*)p);
}

__device__ __forceinline__ int lds_opaque(int v) {
  asm volatile("" : "+v"(v));
  return v;
}

// LDS bank rules on gfx950 (measured with the bank-conflict counter): 64
// banks of 4 bytes.  An 8-byte read serves 32 consecutive lanes per cycle; a
// transposing 8-byte read also serves 32 consecutive lanes but claims banks in
// 32-byte granules; a 16-byte read serves 16 lanes per cycle, the four 4-lane
// quads of a half-wave whose quad index (lane >> 2 & 7) has the same parity.
//
// Swizzle key of token t in a bf16 latent stage: 16-byte chunk c of the
// token's 1 KiB row sits in slot c ^ bf16_key(t).  With the key t & 15 the key
// reads (token t & 15 and chunk group lane >> 4 by lane) are conflict free
// and the transposing value reads are 2-way conflicted; keys that make both
// conflict free exist (for instance ((t & 3) << 1) | (t >> 2 & 1) |
// ((t >> 2 ^ t >> 3) & 1) << 3) but measured slower in this kernel, whose
// LDS traffic is not the limit.
__device__ __forceinline__ int bf16_key(int t) { return t & 15; }

// Swizzle keys of an fp8 stage (e4m3 codes as 512-byte latent rows and 64-byte
// RoPE rows): 16-byte chunk c of latent row t sits in slot c ^ fp8_key(t),
// chunk c of RoPE row t in slot c ^ fp8_rope_key(t).  The key reads (8 bytes,
// 32 lanes per cycle: 16 tokens x both halves of one chunk) and the
// transposing value reads (8 tokens {4G..4G+3, 16+4G..+3} per 16-lane group G,
// 16 tokens per 32 lanes) then touch 16 distinct 16-byte bank groups, and the
// RoPE key reads 16 distinct ones as well.
__device__ __forceinline__ int fp8_key(int t) { return (t & 7) | ((((t >> 3) ^ (t >> 4)) & 1) << 3); }
__device__ __forceinline__ int fp8_rope_key(int t) { return (t >> 2) & 3; }

// Load j of the direct-to-LDS loads of pool block b into a stage
// (Layout::kLoads 1 KiB loads per wave per block).
//   bf16: load j < 16 of wave w is latent row t = 16w + j (lane loads chunk
//         lane ^ bf16_key(t) of the row); loads 16, 17 are RoPE rows
//         16w .. 16w+7 and 16w+8 .. 16w+15 (chunk c in slot c ^ ((t >> 1) & 7)).
//   fp8:  load j < 8 of wave w holds latent rows 2k, 2k+1 (k = 8w + j; lane ->
//         row 2k + (lane >> 5), slot lane & 31, chunk slot ^ fp8_key(row));
//         load 8 holds RoPE rows 16w .. 16w+15 (lane -> row 16w + (lane >> 2),
//         slot lane & 3, chunk slot ^ fp8_rope_key(row)).
template <bool FP8>
__device__ __forceinline__ void issue_load(const PartialParams& p, int b_in, LDS uint8_t* buf,
                                           int wave, int lane_in, int j) {
  using Ly = Layout<FP8>;
  // the block id is the same in every lane; in scalar registers, the pool
  // addresses below are scalar bases
  const int64_t b = __builtin_amdgcn_readfirstlane(b_in);
  // Recompute the per-lane source offsets at every issue instead of letting
  // them be hoisted out of the main loop: registers are scarce there.
  int lane;
  asm volatile("v_mov_b32 %0, %1" : "=v"(lane) : "v"(lane_in));
  const uint8_t* ckv = p.ckv + b * Ly::kStageCkv;
  const uint8_t* kpe = p.kpe + b * (Ly::kStage - Ly::kStageCkv);
  if constexpr (!FP8) {
    if (j < 16) {
      const int t = wave * 16 + j;
      dma16s(ckv + t * 1024, ((uint32_t)lane << 4) ^ (uint32_t)(bf16_key(t) << 4), buf + t * 1024);
    } else {
      const int k = wave * 2 + (j - 16);  // 1 KiB = RoPE rows 8k .. 8k+7
      const int t = 8 * k + (lane >> 3);
      const int c = (lane & 7) ^ ((t >> 1) & 7);
      dma16(kpe + t * 128 + (c << 4), buf + Ly::kStageCkv + k * 1024);
    }
  } else {
    if (j < 8) {
      const int k = wave * 8 + j;
      const int t = 2 * k + (lane >> 5);
      const uint32_t c = (uint32_t)((lane & 31) ^ fp8_key(t));
      dma16s(ckv, (uint32_t)t * 512u + (c << 4), buf + k * 1024);
    } else {
      const int t = 16 * wave + (lane >> 2);
      const uint32_t c = (uint32_t)((lane & 3) ^ fp8_rope_key(t));
      dma16s(kpe, (uint32_t)t * 64u + (c << 4), buf + Ly::kStageCkv + wave * 1024);
    }
  }
}

// All loads of pool block b into a stage.
template <bool FP8>
__device__ __forceinline__ void issue_stage(const PartialParams& p, int b, LDS uint8_t* buf,
                                            int wave, int lane) {
#pragma unroll
  for (int j = 0; j < Layout<FP8>::kLoads; ++j) issue_load<FP8>(p, b, buf, wave, lane, j);
}

// The bf16 loads of one block with their per-block parts precomputed: the
// scalar pool bases and LDS base of this wave's rows, and the lane's byte
// offset.  Latent load j reads row t = 16w + j, whose key bf16_key(t) = j, at
// lane offset (lane16 ^ j << 4) + j * 1024 = lane16 ^ (j << 4 | j << 10).
struct Bf16Issue {
  const uint8_t* ckv;  // row 16w of the block
  const uint8_t* kpe;  // RoPE rows of the block
  uint32_t m0;         // LDS address of row 16w of the stage
  uint32_t lds_rope;   // LDS address of the stage's RoPE part + 2 KiB * w
  __device__ __forceinline__ void load(const PartialParams& p, int j, int wave, int lane_in) const {
    if (j < 16) {
      const uint32_t off = ((uint32_t)lds_opaque(lane_in) << 4) ^ (uint32_t)((j << 4) | (j << 10));
      asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                   :: "v"(off), "s"(ckv), "s"(m0 + (uint32_t)j * 1024u) : "memory", "m0");
    } else {
      int lane;
      asm volatile("v_mov_b32 %0, %1" : "=v"(lane) : "v"(lane_in));
      const int k = wave * 2 + (j - 16);
      const int t = 8 * k + (lane >> 3);
      const int c = (lane & 7) ^ ((t >> 1) & 7);
      const uint32_t d = __builtin_amdgcn_readfirstlane(lds_rope + (uint32_t)(j - 16) * 1024u);
      asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                   :: "v"((uint32_t)(t * 128 + (c << 4))), "s"(kpe), "s"(d) : "memory", "m0");
    }
  }
};

// The bf16 loads of a virtual block of 64 listed tokens (token selections),
// into the same stage layout as a pool block: latent load j of wave w is the
// 1 KiB row of the stage's token 16w + j, read from that token's row of the
// pool (a scalar base per load); RoPE loads 16, 17 are the stage's tokens
// 16w .. 16w+7 and 16w+8 .. 16w+15, a per-lane address each.
struct TokIssue {
  int tok;             // pool token (block * 64 + t) of stage token 16w + (lane & 15)
  uint32_t m0;         // LDS address of row 16w of the stage
  uint32_t lds_rope;   // LDS address of the stage's RoPE part + 2 KiB * w
  __device__ __forceinline__ void load(const PartialParams& p, int j, int wave, int lane_in) const {
    if (j < 16) {
      const uint32_t t = (uint32_t)__builtin_amdgcn_readlane(tok, j);
      const uint8_t* row = p.ckv + (uint64_t)t * 1024u;
      const uint32_t off = ((uint32_t)lds_opaque(lane_in) << 4) ^ (uint32_t)(j << 4);
      asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                   :: "v"(off), "s"(row), "s"(m0 + (uint32_t)j * 1024u) : "memory", "m0");
    } else {
      int lane;
      asm volatile("v_mov_b32 %0, %1" : "=v"(lane) : "v"(lane_in));
      const int src = 8 * (j - 16) + (lane >> 3);  // the lane's token among the wave's 16
      const int t = __shfl(tok, src);
      const int row = 16 * wave + src;             // its row in the stage (swizzle key)
      const int c = (lane & 7) ^ ((row >> 1) & 7);
      const uint8_t* a = p.kpe + (uint64_t)(uint32_t)t * 128u + (uint32_t)(c << 4);
      const uint32_t d = __builtin_amdgcn_readfirstlane(lds_rope + (uint32_t)(j - 16) * 1024u);
      asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                   :: "v"(a), "s"(d) : "memory", "m0");
    }
  }
};

// The fp8 loads of a virtual block of 64 listed tokens, into the same stage
// layout as a pool block (see issue_load): latent load j < 8 of wave w holds
// the stage's tokens 16w + 2j and 16w + 2j + 1 (lanes 0-31 and 32-63), load
// 8 the RoPE rows of tokens 16w .. 16w+15; every lane has its own address.
struct TokIssue8 {
  int tok;       // pool token of stage token 16w + (lane & 15)
  uint32_t buf;  // LDS address of the stage
  __device__ __forceinline__ void load(const PartialParams& p, int j, int wave, int lane_in) const {
    int lane;
    asm volatile("v_mov_b32 %0, %1" : "=v"(lane) : "v"(lane_in));
    const uint8_t* a;
    uint32_t d;
    if (j < 8) {
      const int src = 2 * j + (lane >> 5);
      const int t = 16 * wave + src;
      const uint32_t c = (uint32_t)((lane & 31) ^ fp8_key(t));
      a = p.ckv + (uint64_t)(uint32_t)__shfl(tok, src) * 512u + (c << 4);
      d = buf + (uint32_t)(8 * wave + j) * 1024u;
    } else {
      const int src = lane >> 2;
      const int t = 16 * wave + src;
      const uint32_t c = (uint32_t)((lane & 3) ^ fp8_rope_key(t));
      a = p.kpe + (uint64_t)(uint32_t)__shfl(tok, src) * 64u + (c << 4);
      d = buf + (uint32_t)Layout<true>::kStageCkv + (uint32_t)wave * 1024u;
    }
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :: "v"(a), "s"(__builtin_amdgcn_readfirstlane(d)) : "memory", "m0");
  }
};

// Wait until at most `stages` later stages of this wave's loads are in flight.
template <bool FP8>
__device__ __forceinline__ void wait_stages(int stages) {
  constexpr int L = Layout<FP8>::kLoads;
  if (stages >= 2)
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(2 * L));
  else if (stages == 1)
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(L));
  else
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
}

// Two e4m3 codes (bytes 2*HI, 2*HI+1 of w) -> two bf16, exactly (every e4m3
// value is a bf16 value; the conversion's own scale is 1).
template <bool HI>
__device__ __forceinline__ uint32_t e4m3x2_bf16(uint32_t w) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, HI));
}

// Eight e4m3 codes (two dwords, byte order) -> eight bf16 in the same order.
__device__ __forceinline__ bf16x8_t e4m3x8_bf16(uint32_t w0, uint32_t w1) {
  return __builtin_bit_cast(bf16x8_t, u32x4_t{e4m3x2_bf16<false>(w0), e4m3x2_bf16<true>(w0),
                                              e4m3x2_bf16<false>(w1), e4m3x2_bf16<true>(w1)});
}

// Value fragments of O^T += V^T . P^T from a bf16 tile: fragment f = 32ps + dt
// (k-step ps, column tile dt) must list, for lane (g = lane >> 4, c = lane &
// 15), column 16dt + c of the tokens 32ps + {4g..4g+3, 16+4g..16+4g+3}, in that
// order (the token order of P^T as the S^T products leave it).  Transposing
// 16-bit reads of 4 tokens x 4 columns per lane group of 4: lane (x = lane >> 2,
// q4 = lane & 3) supplies token 32ps + 16hh + x, columns 16dt + 4q4 .. +3 =
// half (q4 & 1) of chunk 2dt + (q4 >> 1), which sits in slot
// (2dt + (q4 >> 1)) ^ bf16_key(x) = 2dt ^ ((q4 >> 1) ^ bf16_key(x)).
struct VFrags {
  const LDS uint8_t* cb;
  int tr_base;
  __device__ __forceinline__ VFrags(const LDS uint8_t* cb_, int lv) : cb(cb_) {
    const int x = lv >> 2, q4 = lv & 3;
    tr_base = x * 1024 + (((q4 >> 1) ^ bf16_key(x)) << 4) + ((q4 & 1) << 3);
  }
  __device__ __forceinline__ bf16x8_t load(int f) const {
    const int ps = f >> 5, dt = f & 31;
    const int o = ps * 32768 + (tr_base ^ (dt << 5));
    const i16x4_t lo = lds_tr16(cb + o);
    const i16x4_t hi = lds_tr16(cb + o + 16384);
    return __builtin_bit_cast(bf16x8_t,
                              i16x8_t{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
  }
};

// Value fragments from an fp8 stage: the same operand as VFrags, read with
// the transposing 8-bit read (each 16-lane group reads 8 tokens x 16 columns;
// lane i = 2r + q supplies token row r, bytes 8q .. 8q+7 of chunk dt) and
// converted to bf16 in registers.  Token row r of group G is
// tb = 4G + r (r < 4) or 16 + 4G + r - 4 of the k-step's 32 tokens, and
// fp8_key(32ps + tb) = fp8_key(tb).
struct VFrags8 {
  const LDS uint8_t* cb;
  int base;
  __device__ __forceinline__ VFrags8(const LDS uint8_t* cb_, int lv) : cb(cb_) {
    const int G = lv >> 4, i = lv & 15, r = i >> 1, q = i & 1;
    const int tb = r < 4 ? 4 * G + r : 16 + 4 * G + (r - 4);
    base = tb * 512 + 8 * q + (fp8_key(tb) << 4);
  }
  __device__ __forceinline__ i32x2_t raw(int f) const {
    const int ps = f >> 5, dt = f & 31;
    return __builtin_bit_cast(
        i32x2_t, __builtin_amdgcn_ds_read_tr8_b64_v2i32((LDS i32x2_t*)(cb + ps * 16384 + (base ^ (dt << 4)))));
  }
};

// The score factors of an fp8 block with latent scale sc and RoPE scale sk.
// Its scores are scale * (sc * (q_lat . latent codes) + sk * (q_pe . RoPE
// codes)); the kernel forms them as main * (q_lat . latent codes + ratio *
// (q_pe . RoPE codes)), one accumulator for both parts.  While |sk| < 2^64 |sc|
// that is exact: main = sc, ratio = sk / sc.  Otherwise (a latent scale of 0,
// or one below 2^-64 of the RoPE scale) main = sk * 2^-64 and ratio = 2^64:
// the score then differs from the exact one by (sk 2^-64 - sc)(q_lat . codes),
// at most 2^-63 |sk| |q_lat . codes|, and nothing is divided by zero.  The
// values themselves always take the latent scale sc.
__device__ __forceinline__ void fp8_factors(float sc, float sk, float& main, float& ratio) {
  constexpr float kBig = 18446744073709551616.0f;  // 2^64
  if (fabsf(sk) < kBig * fabsf(sc)) {
    main = sc;
    ratio = sk / sc;
  } else {
    main = sk * (1.0f / kBig);
    ratio = kBig;
  }
}

// Per-listed-block fp8 factors in LDS: [3 i] value scale, [3 i + 1] score
// factor main, [3 i + 2] RoPE ratio (see fp8_factors).
__device__ __forceinline__ void put_fp8_factors(LDS float* scales, int i, float sc, float sk) {
  float main, ratio;
  fp8_factors(sc, sk, main, ratio);
  scales[3 * i] = sc;
  scales[3 * i + 1] = main;
  scales[3 * i + 2] = ratio;
}

// Compact the valid selected blocks of slots [slot0, slot0 + nslots) of job r
// into the LDS list (slot order kept); for fp8 also each listed block's
// factors (put_fp8_factors).  first_id: the id of slot slot0 + tid, already
// loaded (see first_slot_id).  Returns the number of listed blocks.
template <bool FP8>
__device__ __forceinline__ int compact_slots(const PartialParams& p, int r, int slot0, int nslots,
                                             int first_id, LDS uint8_t* smem, int tid) {
  using L = Layout<FP8>;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  LDS int* list = (LDS int*)(smem + L::kList);
  LDS float* scales = (LDS float*)(smem + L::kScales);
  LDS int* wave_cnt = (LDS int*)(smem + L::kWaveCnt);
  int n_valid = 0;
  for (int base = 0; base < nslots; base += 256) {
    const int i = base + tid;
    int b = -1;
    if (i < nslots) {
      const int id = base == 0 ? first_id : p.sel[r * p.sel_s0 + slot0 + i];
      if (id >= 0 && id < p.NB) {
        const int bb = p.table[r * p.table_s0 + id];
        if (bb >= 0 && bb < p.P) b = bb;
      }
    }
    const uint64_t m = __ballot(b >= 0);
    const int before = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) wave_cnt[wave] = __popcll(m);
    lds_barrier();
    int off = n_valid, total = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const int c = wave_cnt[w];
      off += (w < wave) ? c : 0;
      total += c;
    }
    if (b >= 0) {
      list[off + before] = b;
      if constexpr (FP8) put_fp8_factors(scales, off + before, p.ckv_scale[b], p.kpe_scale[b]);
    }
    n_valid += total;
    lds_barrier();
  }
  return n_valid;
}

// Per-row selections: compact the blocks that query rows i0 .. i0 + n_i - 1
// of job r select in slots [slot0, slot0 + nslots), among the logical blocks
// id0, id0 + id_step, id0 + 2 id_step, ... below NB, into the LDS list, each
// block once per copy, with a mask of the rows that hold that copy: a block
// that row i lists c_i times gives max_i c_i entries, entry k carrying the
// rows with c_i > k.  Each row thus attends exactly its own multiset, and a
// block that several rows chose is loaded once for all of them.  Entries
// come in ascending logical-block order.  The counters (16 bits per (block,
// row) of the blocks taken; at most nslots each) use the stage area, which is
// free until the first load is issued.  Returns the number of entries.
// fp8: each entry also gets its block's factors (put_fp8_factors).
// first_id: the id of this thread's first entry (row i0 + tid / nslots, slot
// slot0 + tid % nslots), already loaded.
template <bool FP8>
__device__ __forceinline__ int compact_per_row(const PartialParams& p, int r, int slot0,
                                               int nslots, int id0, int id_step, int i0, int n_i,
                                               int first_id, LDS uint8_t* smem, LDS int* list,
                                               LDS uint64_t* masks, int tid) {
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  LDS uint32_t* cnt = (LDS uint32_t*)smem;
  LDS const uint16_t* cnt16 = (LDS const uint16_t*)smem;
  LDS int* wave_cnt = (LDS int*)(smem + Layout<FP8>::kWaveCnt);
  LDS float* scales = (LDS float*)(smem + Layout<FP8>::kScales);
  const int n_ids = id0 < p.NB ? (p.NB - id0 + id_step - 1) / id_step : 0;
  const int n_words = (n_ids * n_i + 1) >> 1;
  for (int w = tid; w < n_words; w += 256) cnt[w] = 0u;
  lds_barrier();
  const int n_ent = n_i * nslots;
  for (int e = tid; e < n_ent; e += 256) {
    const int ii = e / nslots, j = e - ii * nslots;
    const int id = e == tid ? first_id : p.sel[r * p.sel_s0 + (int64_t)(i0 + ii) * p.sel_s1 + slot0 + j];
    const int u = (id - id0) / id_step;
    if (id >= id0 && id < p.NB && u * id_step == id - id0) {
      const int bb = p.table[r * p.table_s0 + id];
      if (bb >= 0 && bb < p.P) {
        const int c = u * n_i + ii;
        __atomic_fetch_add(&cnt[c >> 1], 1u << ((c & 1) * 16), __ATOMIC_RELAXED);
      }
    }
  }
  lds_barrier();
  int n_valid = 0;
  for (int base = 0; base < n_ids; base += 256) {
    const int u = base + tid, id = id0 + u * id_step;
    int kmax = 0;
    if (u < n_ids)
      for (int ii = 0; ii < n_i; ++ii) kmax = max(kmax, (int)cnt16[u * n_i + ii]);
    // exclusive prefix sum of kmax over the workgroup (ascending id)
    int incl = kmax;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int v = __shfl_up(incl, o);
      if (lane >= o) incl += v;
    }
    if (lane == 63) wave_cnt[wave] = incl;
    lds_barrier();
    int off = n_valid + incl - kmax, total = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const int c = wave_cnt[w];
      off += (w < wave) ? c : 0;
      total += c;
    }
    if (kmax > 0) {
      const int bb = p.table[r * p.table_s0 + id];
      float sc = 1.f, sk = 1.f;
      if constexpr (FP8) {
        sc = p.ckv_scale[bb];
        sk = p.kpe_scale[bb];
      }
      for (int k = 0; k < kmax; ++k) {
        uint64_t m = 0;
        for (int ii = 0; ii < n_i; ++ii)
          if ((int)cnt16[u * n_i + ii] > k) m |= 1ull << ii;
        list[off + k] = bb;
        masks[off + k] = m;
        if constexpr (FP8) put_fp8_factors(scales, off + k, sc, sk);
      }
    }
    n_valid += total;
    lds_barrier();
  }
  return n_valid;
}

// Token selections: compact the valid token ids of slots [slot0, slot0 +
// nslots) of job r into the LDS list as pool tokens (table[r, id / 64] * 64 +
// id % 64), slot order kept, and fill the list up to the next multiple of 64
// with the first entry, so that the last virtual block loads only listed
// tokens (the fill is masked out of the softmax).  first_id as for
// compact_slots.  fp8: each token carries
// its own block's factors (fp8_factors): the value scale in tok_scales[i],
// the RoPE ratio in tok_scales[kMaxSlotsPerSplit + i] and the score factor
// in tok_scales[2 kMaxSlotsPerSplit + i].  Returns the number of listed
// tokens.
template <bool FP8>
__device__ __forceinline__ int compact_tokens(const PartialParams& p, int r, int slot0,
                                              int nslots, int first_id, LDS uint8_t* smem,
                                              int tid) {
  using L = Layout<FP8>;
  LDS float* tok_scales = (LDS float*)(smem + L::kScales);
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  LDS int* list = (LDS int*)(smem + L::kList);
  LDS int* wave_cnt = (LDS int*)(smem + L::kWaveCnt);
  const int64_t n_ids = (int64_t)p.NB * kBlock;
  int n_tok = 0;
  for (int base = 0; base < nslots; base += 256) {
    const int i = base + tid;
    int pt = -1;
    if (i < nslots) {
      const int id = base == 0 ? first_id : p.sel[r * p.sel_s0 + slot0 + i];
      if (id >= 0 && id < n_ids) {
        const int bb = p.table[r * p.table_s0 + (id >> 6)];
        if (bb >= 0 && bb < p.P) pt = bb * kBlock + (id & (kBlock - 1));
      }
    }
    const uint64_t m = __ballot(pt >= 0);
    const int before = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) wave_cnt[wave] = __popcll(m);
    lds_barrier();
    int off = n_tok, total = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const int c = wave_cnt[w];
      off += (w < wave) ? c : 0;
      total += c;
    }
    if (pt >= 0) {
      list[off + before] = pt;
      if constexpr (FP8) {
        const int bb = pt >> 6;
        const float sc = p.ckv_scale[bb];
        float main, ratio;
        fp8_factors(sc, p.kpe_scale[bb], main, ratio);
        tok_scales[off + before] = sc;
        tok_scales[kMaxSlotsPerSplit + off + before] = ratio;
        tok_scales[2 * kMaxSlotsPerSplit + off + before] = main;
      }
    }
    n_tok += total;
    lds_barrier();
  }
  const int padded = (n_tok + kBlock - 1) & ~(kBlock - 1);
  for (int i = tid; i < padded; i += 256) {
    if (i >= n_tok) {
      list[i] = list[0];
      if constexpr (FP8) {
        tok_scales[i] = tok_scales[0];
        tok_scales[kMaxSlotsPerSplit + i] = tok_scales[kMaxSlotsPerSplit];
        tok_scales[2 * kMaxSlotsPerSplit + i] = tok_scales[2 * kMaxSlotsPerSplit];
      }
    }
  }
  lds_barrier();
  return n_tok;
}

// RG row groups of 16 per wave: wave w computes rows 16*RG*w .. 16*RG*(w+1)-1
// of the row tile (64*RG rows) over all 512 latent columns.  KV is the cache
// kind: bf16, e4m3 with one scale per block for the whole 576-wide entries, or
// e4m3 with separate latent and RoPE scales per block.
template <int RG, int KV, int SEL>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void partial_kernel(const PartialParams p) {
  constexpr bool FP8 = KV != kKvBf16;
  constexpr bool PR = SEL == kSelPerRow;   // a block selection per query row
  constexpr bool TOK = SEL == kSelTokens;  // token selections, 64 to a virtual block
  constexpr bool kSplitScales = KV == kKvFp8Split;
  using L = Layout<FP8>;
  constexpr int kTau4 = kBlock / 16;   // 16-token tiles per block
  constexpr int kKSteps = kBlock / 32;  // 32-token PV k-steps per block
  constexpr int kRowsWg = 64 * RG;
  __shared__ __attribute__((aligned(16))) uint8_t smem_raw[PR ? L::kTotalPerRow : L::kTotal];
  LDS uint8_t* smem = (LDS uint8_t*)smem_raw;
  LDS uint8_t* const stage0 = smem;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n16 = lane & 15;  // MFMA column / row-in-group index
  const int g = lane >> 4;    // MFMA k-group

  // ---- work item.  Workgroups go to the 8 XCDs round-robin; the ids are
  // renumbered so that each XCD takes one contiguous range.  The splits of a
  // row tile then run on one XCD, and the combine, renumbered alike, reads
  // their rows on that XCD when both grids split the rows alike.  Per-row
  // selections split by logical block over many row tiles are numbered the
  // other way round (row tiles fastest): every tile's split s reads blocks
  // of the same residue class, which then meet in the L2 of one or two XCDs
  // instead of all eight (the query rows, read once per split, are what is
  // fetched more than once instead, the smaller of the two).
  const int w_id = gridDim.x % 8 ? (int)blockIdx.x
                                 : (int)(blockIdx.x % 8) * (int)(gridDim.x / 8) + (int)(blockIdx.x / 8);
  const bool tiles_fast = PR && p.tiles_fast;
  const int s_idx = tiles_fast ? (w_id / p.row_tiles) % p.n_splits : w_id % p.n_splits;
  const int rt = tiles_fast ? w_id % p.row_tiles : (w_id / p.n_splits) % p.row_tiles;
  const int r_num = w_id / (p.n_splits * p.row_tiles);
  // jobs that share q rows (r, r + q_jobs, ...) take consecutive numbers
  const int r = p.q_rep > 1 ? (r_num % p.q_rep) * p.q_jobs + r_num / p.q_rep : r_num;
  const int rq = r % p.q_jobs;  // the job's q rows
  const int slot0 = s_idx * p.slots_per_split;
  const int nslots = max(0, min(p.K - slot0, p.slots_per_split));

  // ---- prologue.  Three dependent trips to memory (slot ids, block table,
  // then the first blocks) come before the first product; the query rows go
  // out between the first two, so that their latency hides behind the
  // compaction's.
  LDS int* list = (LDS int*)(smem + L::kList);
  LDS float* scales = (LDS float*)(smem + L::kScales);
  LDS uint64_t* masks = (LDS uint64_t*)(smem + L::kMasks);
  const int i0 = rt * kRowsWg / p.H;  // first query row of the tile
  // per-row selections: the query rows of the tile; split by logical block
  // (split s takes blocks s, s + S, ... from every slot), so that rows which
  // chose one block in different slots share its load, or by slot range when
  // a tile's slots may not fit one list
  const int n_i = PR ? (min((rt + 1) * kRowsWg, p.rows) - 1) / p.H - i0 + 1 : 1;
  const int c_slot0 = PR && p.split_by_id ? 0 : slot0;
  const int c_nslots = PR && p.split_by_id ? p.K : nslots;
  // the slot id this thread compacts first
  int first_id = -1;
  if constexpr (PR) {
    if (tid < n_i * c_nslots) {
      const int ii = tid / c_nslots, j = tid - ii * c_nslots;
      first_id = p.sel[r * p.sel_s0 + (int64_t)(i0 + ii) * p.sel_s1 + c_slot0 + j];
    }
  } else {
    if (tid < nslots) first_id = p.sel[r * p.sel_s0 + slot0 + tid];
  }

  // this wave's query rows as MFMA B operands, held for the whole kernel:
  // k-step ks (0..15 latent, 16..17 RoPE) covers 32 dims, lane group g takes
  // dims 32ks' + 8g .. +7 (ks' = the step within its part).
  const int row_wg0 = rt * kRowsWg;
  bf16x8_t qb[RG][18];
#pragma unroll
  for (int rg = 0; rg < RG; ++rg) {
    const int row = row_wg0 + wave * 16 * RG + rg * 16 + n16;
    if (row < p.rows) {
      const int i = row / p.H, h = row - (row / p.H) * p.H;
      const uint16_t* ql = p.q_lat + rq * p.ql_s0 + i * p.ql_s1 + h * p.ql_s2 + g * 8;
      const uint16_t* qp = p.q_pe + rq * p.qp_s0 + i * p.qp_s1 + h * p.qp_s2 + g * 8;
#pragma unroll
      for (int ks = 0; ks < 16; ++ks) qb[rg][ks] = *(const bf16x8_t*)(ql + ks * 32);
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) qb[rg][16 + ks] = *(const bf16x8_t*)(qp + ks * 32);
    } else {
#pragma unroll
      for (int ks = 0; ks < 18; ++ks) qb[rg][ks] = bf16x8_t{};
    }
  }

  // compact the valid selected blocks of the slot range (slot order kept;
  // per-row selections: the union over the tile's query rows, with row masks)
  int n_valid;
  int n_tok = 0;  // token selections: the listed tokens (n_valid counts virtual blocks)
  if constexpr (PR) {
    n_valid = compact_per_row<FP8>(p, r, c_slot0, c_nslots, p.split_by_id ? s_idx : 0,
                                   p.split_by_id ? p.n_splits : 1, i0, n_i, first_id, smem, list,
                                   masks, tid);
  } else if constexpr (TOK) {
    n_tok = compact_tokens<FP8>(p, r, slot0, nslots, first_id, smem, tid);
    n_valid = (n_tok + kBlock - 1) / kBlock;
  } else {
    n_valid = compact_slots<FP8>(p, r, slot0, nslots, first_id, smem, tid);
  }

  // the first blocks' loads
  if constexpr (TOK && FP8) {
    for (int h = 0; h < n_valid && h < L::kLead; ++h) {
      TokIssue8 ti;
      ti.tok = list[h * kBlock + 16 * wave + (lane & 15)];
      ti.buf = (uint32_t)(uintptr_t)(stage0 + h * L::kStage);
#pragma unroll
      for (int j = 0; j < L::kLoads; ++j) ti.load(p, j, wave, lane);
    }
  } else if constexpr (TOK) {
    static_assert(L::kLead == 1, "bf16 token selections stream one virtual block ahead");
    if (n_valid > 0) {
      TokIssue ti;
      ti.tok = list[16 * wave + (lane & 15)];
      ti.m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)stage0 + (uint32_t)wave * 16384u);
      ti.lds_rope = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)stage0 + 65536u + (uint32_t)wave * 2048u);
#pragma unroll
      for (int j = 0; j < L::kLoads; ++j) ti.load(p, j, wave, lane);
    }
  } else {
    for (int h = 0; h < n_valid && h < L::kLead; ++h)
      issue_stage<FP8>(p, list[h], stage0 + h * L::kStage, wave, lane);
  }
  // Q (and with it the first stages) is resident before the main loop, so
  // that the only vector-memory operations in flight inside the loop are the
  // prefetches the loop issues itself.
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));

  f32x4_t O[32][RG];
#pragma unroll
  for (int dt = 0; dt < 32; ++dt)
#pragma unroll
    for (int rg = 0; rg < RG; ++rg) O[dt][rg] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run[RG], l_run[RG];
  // the largest score of each row so far (log2 units): the wire form's m
  float m_true[RG];
  // per-row selections: the bit of each of the lane's rows in the entry masks
  // (rows past the end of the job are never stored; any bit will do)
  int row_bit[RG];
#pragma unroll
  for (int rg = 0; rg < RG; ++rg) {
    const int row = row_wg0 + wave * 16 * RG + rg * 16 + n16;
    row_bit[rg] = PR ? min(max(row / p.H - i0, 0), 63) : 0;
  }
#pragma unroll
  for (int rg = 0; rg < RG; ++rg) {
    m_run[rg] = -INFINITY;
    l_run[rg] = 0.f;
    m_true[rg] = -INFINITY;
  }

  // ---- main loop over the listed blocks; L::kLead blocks stream in while one
  // is computed
  for (int h = 0; h < n_valid; ++h) {
    wait_stages<FP8>(min(n_valid - 1 - h, L::kLead - 1));
    lds_barrier();  // block h is in LDS for every wave; every wave is done with block h-1
    // The pool block that streams into the stage freed by this block (read
    // from LDS first: LDS reads complete in order).
    const int hn = h + L::kLead;
    const int b_next = hn >= n_valid ? -1 : TOK ? 0 : __builtin_amdgcn_readfirstlane(list[hn]);
    uint64_t emask = ~0ull;  // the rows this entry is attended by
    if constexpr (PR) {
      // (readfirstlane returns int: widen through uint32_t, not by sign)
      const uint64_t m = masks[h];
      const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(m >> 32));
      const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)m);
      emask = ((uint64_t)hi << 32) | (uint64_t)lo;
    }
    __builtin_amdgcn_sched_barrier(0);
    // fp8: the scores are accumulated as ratio * (q_pe . kpe codes) +
    // q_lat . ckv codes and then scaled by the softmax scale times the
    // block's score factor (fp8_factors); P is scaled by the latent scale
    // before its bf16 rounding.
    float s_mult = p.scale_log2, v_mult = 1.f, pe_ratio = 1.f;
    if constexpr (FP8 && !TOK) {
      v_mult = scales[3 * h];
      if constexpr (kSplitScales) pe_ratio = scales[3 * h + 2];
      s_mult = p.scale_log2 * scales[3 * h + 1];
    }
    const LDS uint8_t* const cb = stage0 + (h % L::kNum) * L::kStage;
    // The next stage's loads.  bf16: two per S^T step over the first nine
    // steps, beside the products, with the per-block address parts computed
    // once (all 18 at once would hold the four waves for about 1.6k cycles at
    // the per-CU address unit, which takes one 1 KiB load per ~16 cycles).
    // fp8 (9 loads): one per two S^T steps.
    LDS uint8_t* const next_buf = stage0 + (hn % L::kNum) * L::kStage;
    typename std::conditional<TOK, TokIssue, Bf16Issue>::type bi;
    if constexpr (TOK && !FP8) {
      bi.tok = b_next >= 0 ? list[hn * kBlock + 16 * wave + (lane & 15)] : 0;
      bi.m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)next_buf + (uint32_t)wave * 16384u);
      bi.lds_rope = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)next_buf + 65536u + (uint32_t)wave * 2048u);
    } else if constexpr (!FP8) {
      const int64_t bn = b_next >= 0 ? b_next : 0;
      bi.ckv = p.ckv + bn * 65536 + wave * 16384;
      bi.kpe = p.kpe + bn * 8192;
      bi.m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)next_buf + (uint32_t)wave * 16384u);
      bi.lds_rope = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)next_buf + 65536u + (uint32_t)wave * 2048u);
    }
    // Per-lane LDS offsets are recomputed from an opaque copy of the lane id in
    // every iteration (a few VALU ops) rather than held in registers across
    // the loop.
    const int ln = lds_opaque(lane);
    const int ln16 = ln & 15, lg = ln >> 4;
    // fp8 token selections: the per-token scales of the lane's S^T elements
    // (tokens 16 tau + 4 lg + k), read from LDS where they are used so that
    // they hold no registers across the products
    LDS const float* const tok_scales = (LDS const float*)(smem + L::kScales);
    auto tok_scale4 = [&](int which, int tau) -> f32x4_t {
      return *(LDS const f32x4_t*)(tok_scales + which * kMaxSlotsPerSplit + h * kBlock +
                                   16 * tau + 4 * lg);
    };

    // S^T[token][row] for tokens 16*tau + ln16: 18 k-steps (2 RoPE, then 16
    // latent), 4 token tiles each.  Software pipeline: key fragments are
    // requested about two steps before their products; the scheduling fences
    // keep the compiler from regrouping loads next to their use.
    f32x4_t sacc[RG][kTau4];
    {
      // bf16: latent chunk 4ks+lg of token 16tau+ln16 sits in slot
      // (4ks+lg) ^ bf16_key(ln16) = 4ks ^ (lg ^ bf16_key(ln16)).
      // fp8: the lane reads 8 codes, bytes 32ks + 8lg .. of the row = half
      // (lg & 1) of chunk 2ks + (lg >> 1), slot (2ks + (lg >> 1)) ^ fp8_key(t)
      // with fp8_key(16tau + n) = fp8_key(n) ^ (tau & 1) << 3; RoPE rows
      // likewise with fp8_rope_key(16tau + n) = fp8_rope_key(n).
      const int key_base = FP8 ? ln16 * 512 + 8 * (lg & 1) + (((lg >> 1) ^ fp8_key(ln16)) << 4)
                               : ln16 * 1024 + ((lg ^ bf16_key(ln16)) << 4);
      const int rope_base = FP8 ? L::kStageCkv + ln16 * 64 + 8 * (lg & 1) +
                                      (((lg >> 1) ^ fp8_rope_key(ln16)) << 4)
                                : L::kStageCkv + ln16 * 128;
      // bf16: the ring holds operands; fp8: it holds codes, converted at use
      using KRing = typename std::conditional<FP8, i32x2_t, bf16x8_t>::type;
      auto key_frags = [&](int step, KRing (&a)[kTau4]) {
        if constexpr (FP8) {
          if (step < 2) {
#pragma unroll
            for (int tau = 0; tau < kTau4; ++tau)
              a[tau] = *(const LDS i32x2_t*)(cb + tau * 1024 + (rope_base ^ (step << 5)));
          } else {
            const int ks = step - 2;
#pragma unroll
            for (int tau = 0; tau < kTau4; ++tau)
              a[tau] = *(const LDS i32x2_t*)(cb + tau * 8192 + (key_base ^ ((ks << 5) ^ ((tau & 1) << 7))));
          }
        } else if (step < 2) {
#pragma unroll
          for (int tau = 0; tau < kTau4; ++tau)
            a[tau] = lds_b128(cb + tau * 2048 + rope_base + (((4 * step + lg) ^ (ln16 >> 1)) << 4));
        } else {
          const int ks = step - 2;
#pragma unroll
          for (int tau = 0; tau < kTau4; ++tau)
            a[tau] = lds_b128(cb + tau * 16384 + (key_base ^ (ks << 6)));
        }
      };
      // bf16: the fragment of one token tile
      auto key_frag = [&](int step, int tau, bf16x8_t& a) {
        if constexpr (!FP8) {
          if (step < 2)
            a = lds_b128(cb + tau * 2048 + rope_base + (((4 * step + lg) ^ (ln16 >> 1)) << 4));
          else
            a = lds_b128(cb + tau * 16384 + (key_base ^ ((step - 2) << 6)));
        }
      };
      auto key_ops = [&](const KRing (&r)[kTau4], bf16x8_t (&a)[kTau4]) {
#pragma unroll
        for (int tau = 0; tau < kTau4; ++tau) {
          if constexpr (FP8) a[tau] = e4m3x8_bf16((uint32_t)r[tau][0], (uint32_t)r[tau][1]);
          else a[tau] = r[tau];
        }
      };
      // Codes are converted one step before their products: a VALU write of
      // an operand is not interlocked against the products that read it, and
      // a whole group of products lies between the two.  The first step's
      // group leads with the wait states instead.
      KRing kr[3][kTau4];
      bf16x8_t ka[2][kTau4];
      key_frags(0, kr[0]);
      key_frags(1, kr[1]);
      key_ops(kr[0], ka[0]);
#pragma unroll
      for (int step = 0; step < 18; ++step) {
        if (FP8 && step + 2 < 18) key_frags(step + 2, kr[(step + 2) % 3]);
        if constexpr (FP8) {
          // Single products, tile by tile; after the products of tile t the
          // codes of tile t of the next step are converted to bf16 (4 VALU
          // ops beside the matrix core), 3 RG products before the first one
          // that reads them; one load of a later block per two steps.
          __builtin_amdgcn_sched_barrier(0);
          const int ks = step < 2 ? 16 + step : step - 2;
          const bf16x8_t(&a)[kTau4] = ka[step % 2];
          const bool ratio_step = kSplitScales && step == 2;
          if (ratio_step) {
#pragma unroll
            for (int rg = 0; rg < RG; ++rg)
#pragma unroll
              for (int tau = 0; tau < kTau4; ++tau) {
                if constexpr (TOK) scale_inplace4(sacc[rg][tau], tok_scale4(1, tau));
                else scale_inplace(sacc[rg][tau], pe_ratio);
              }
          }
          constexpr int kPer = RG * kTau4;
#pragma unroll
          for (int j = 0; j < kPer; ++j) {
            const int tau = j / RG, rg = j % RG;
            const bf16x8_t q = qb[rg][ks];
            // the RoPE steps end with the wait states the ratio's VALU reads
            // of the results need; the last step with those any read needs
            const bool pad = (step == 17 || (kSplitScales && step == 1)) && j == kPer - 1;
            if (step == 0)
              st1<true, false, true>(sacc[rg][tau], a[tau], q);
            else if (pad)
              st1<false, true, false>(sacc[rg][tau], a[tau], q);
            else if (ratio_step)
              // every product of this step leads with the wait states: the
              // ratio's VALU writes of the accumulators come right before
              st1<false, false, true>(sacc[rg][tau], a[tau], q);
            else
              st1<false, false, false>(sacc[rg][tau], a[tau], q);
            __builtin_amdgcn_sched_barrier(0);
            if (rg == RG - 1 && step + 1 < 18) {
              const KRing& w = kr[(step + 1) % 3][tau];
              bf16x8_t& dst = ka[(step + 1) % 2][tau];
              dst = e4m3x8_bf16((uint32_t)w[0], (uint32_t)w[1]);
              pin(dst);
            }
            if (j == kPer / 2 && (step & 1) == 0 && b_next >= 0) {
              if constexpr (TOK) {
                TokIssue8 ti;
                ti.tok = list[hn * kBlock + 16 * wave + (lane & 15)];
                ti.buf = (uint32_t)(uintptr_t)next_buf;
                ti.load(p, step >> 1, wave, lane);
              } else {
                issue_load<true>(p, b_next, next_buf, wave, lane, step >> 1);
              }
            }
            __builtin_amdgcn_sched_barrier(0);
          }
          continue;
        }
        // bf16: single products, with the key reads of step + 2 (one per
        // token tile) and this step's loads of the next block between them
        if constexpr (!FP8) {
        const int ks = step < 2 ? 16 + step : step - 2;
        constexpr int kPer = RG * kTau4;  // products per step
#pragma unroll
        for (int j = 0; j < kPer; ++j) {
          const int tau = j / RG, rg = j % RG;
          const bf16x8_t a = kr[step % 3][tau];
          if (step == 0)
            st1<true, false>(sacc[rg][tau], a, qb[rg][ks]);
          else if (step == 17 && j == kPer - 1)
            st1<false, true>(sacc[rg][tau], a, qb[rg][ks]);
          else
            st1<false, false>(sacc[rg][tau], a, qb[rg][ks]);
          __builtin_amdgcn_sched_barrier(0);
          // after the products of tile t (RG = 2) or tile t itself (RG = 1):
          // the read of tile t of step + 2; then the two loads
          if (rg == RG - 1 && step + 2 < 18) key_frag(step + 2, tau, kr[(step + 2) % 3][tau]);
          if (step < 9 && b_next >= 0 && j == kPer - 3) bi.load(p, 2 * step, wave, lane);
          if (step < 9 && b_next >= 0 && j == kPer - 2) bi.load(p, 2 * step + 1, wave, lane);
          __builtin_amdgcn_sched_barrier(0);
        }
        }
      }
    }

    // The first value fragments of O^T += V^T . P^T are requested before the
    // softmax, whose VALU work then covers their latency.
    constexpr int kPvAhead = 8;
    constexpr int kFrags = 32 * kKSteps;
    const VFrags vf(cb, lds_opaque(lane));
    const VFrags8 vf8(cb, lds_opaque(lane));
    // bf16: the ring holds operands; fp8: it holds codes (converted at use)
    using VRing = typename std::conditional<FP8, i32x2_t, bf16x8_t>::type;
    auto vload = [&](int f) -> VRing {
      if constexpr (FP8) return vf8.raw(f); else return vf.load(f);
    };
    auto vop = [&](const VRing& x) -> bf16x8_t {
      if constexpr (FP8) return e4m3x8_bf16((uint32_t)x[0], (uint32_t)x[1]); else return x;
    };
    VRing vr[kPvAhead + 1];
#pragma unroll
    for (int f = 0; f < kPvAhead; ++f) vr[f] = vload(f);
    // fp8: operands are converted two fragments ahead, after the products of
    // a fragment, so that the conversion runs beside them and no product waits
    // for a conversion just issued
    bf16x8_t vc[3];
    __builtin_amdgcn_sched_barrier(0);

    f32x4_t acc[RG][kTau4];
#pragma unroll
    for (int rg = 0; rg < RG; ++rg)
#pragma unroll
      for (int tau = 0; tau < kTau4; ++tau) acc[rg][tau] = sacc[rg][tau];

    // Online softmax over the block's 64 tokens (exp2 domain).  Lane (n16, g)
    // holds row n16 of each row group and tokens 16*tau + 4g + i.
    bool need_any = false;
    float bmax[RG];
    // token selections: the listed tokens in this virtual block (the rest of
    // the last one is fill, with no weight)
    const int n_here = TOK ? n_tok - h * kBlock : kBlock;
    // (fp8 token selections: each token's value is code * its block's
    // latent scale, and its score is scaled likewise)
#pragma unroll
    for (int rg = 0; rg < RG; ++rg) {
      float bm = -INFINITY;
#pragma unroll
      for (int tau = 0; tau < kTau4; ++tau) {
        if constexpr (FP8 && TOK) acc[rg][tau] *= tok_scale4(2, tau) * s_mult;
        else acc[rg][tau] *= s_mult;
        if (TOK && n_here < kBlock) {
#pragma unroll
          for (int k = 0; k < 4; ++k)
            if (16 * tau + 4 * lg + k >= n_here) acc[rg][tau][k] = -INFINITY;
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) bm = fmaxf(bm, acc[rg][tau][k]);
      }
      bmax[rg] = xor_max(bm);
      if constexpr (PR) {
        // a row that does not attend this entry: no maximum, no weights
        if (((emask >> row_bit[rg]) & 1ull) == 0) bmax[rg] = -INFINITY;
      }
      m_true[rg] = fmaxf(m_true[rg], bmax[rg]);
      need_any |= bmax[rg] > m_run[rg] + kTau;
    }
    if (__ballot(need_any) != 0) {
#pragma unroll
      for (int rg = 0; rg < RG; ++rg) {
        float alpha = 1.f;
        if (bmax[rg] > m_run[rg] + kTau) {
          if (m_run[rg] != -INFINITY) alpha = __builtin_amdgcn_exp2f(m_run[rg] - bmax[rg]);
          m_run[rg] = bmax[rg];
          l_run[rg] *= alpha;
        }
        if (__ballot(alpha != 1.f) != 0) {
#pragma unroll
          for (int dt = 0; dt < 32; ++dt) O[dt][rg] = scale_acc(O[dt][rg], alpha);
        }
      }
    }
    // P^T B operands: k-step ps covers tokens 32ps + {4g..4g+3, 16+4g..16+4g+3}
    // (token tiles 2ps and 2ps+1).  The row sum takes the unrounded fp32
    // weights; the PV operand is rounded to bf16 (after the latent scale, for
    // fp8).  The weights of k-step 0 are computed here; those of k-step 1 are
    // computed two at a time between the products of k-step 0, which does not
    // need them, so that this VALU work runs beside the matrix core.
    bf16x8_t pb[RG][kKSteps];
    float psum[RG];
    bool on[RG];
#pragma unroll
    for (int rg = 0; rg < RG; ++rg) on[rg] = !PR || ((emask >> row_bit[rg]) & 1ull) != 0;
    auto p_pair = [&](int rg, int tau, int k0) {
      // (an exact 0 for rows that do not attend this entry, also before
      // their first attended entry, when m_run is still -inf)
      float e0 = __builtin_amdgcn_exp2f(acc[rg][tau][k0] - m_run[rg]);
      float e1 = __builtin_amdgcn_exp2f(acc[rg][tau][k0 + 1] - m_run[rg]);
      if constexpr (PR) {
        e0 = on[rg] ? e0 : 0.f;
        e1 = on[rg] ? e1 : 0.f;
      }
      psum[rg] += e0 + e1;
      float vm0 = v_mult, vm1 = v_mult;
      if constexpr (FP8 && TOK) {
        vm0 = tok_scales[h * kBlock + 16 * tau + 4 * lg + k0];
        vm1 = tok_scales[h * kBlock + 16 * tau + 4 * lg + k0 + 1];
      }
      pb[rg][tau >> 1][(tau & 1) * 4 + k0] = (__bf16)(FP8 ? e0 * vm0 : e0);
      pb[rg][tau >> 1][(tau & 1) * 4 + k0 + 1] = (__bf16)(FP8 ? e1 * vm1 : e1);
    };
#pragma unroll
    for (int rg = 0; rg < RG; ++rg) {
      psum[rg] = 0.f;
#pragma unroll
      for (int tau = 0; tau < 2; ++tau) {
        p_pair(rg, tau, 0);
        p_pair(rg, tau, 2);
      }
    }
    // pair i (i < 4 * RG) of k-step 1: row group i >> 2, tile 2 + ((i >> 1) & 1),
    // elements 2 (i & 1) and 2 (i & 1) + 1
    constexpr int kLatePairs = 4 * RG;
    constexpr int kLateStride = 32 / kLatePairs;

    // O^T[dim][row] += V^T . P^T over 2 k-steps x 32 column tiles, in a
    // software pipeline kPvAhead fragments deep.
#pragma unroll
    for (int f = 0; f < kFrags; ++f) {
      if (f + kPvAhead < kFrags) vr[(f + kPvAhead) % (kPvAhead + 1)] = vload(f + kPvAhead);
      if (f < 32 && f % kLateStride == 0) {
        const int i = f / kLateStride;
        p_pair(i >> 2, 2 + ((i >> 1) & 1), 2 * (i & 1));
      }
      __builtin_amdgcn_sched_barrier(0);
      const int ps = f >> 5, dt = f & 31;
      if constexpr (FP8) {
        if (f == 0) {
          vc[0] = vop(vr[0]);
          vc[1] = vop(vr[1]);
        }
#pragma unroll
        for (int rg = 0; rg < RG; ++rg) O[dt][rg] = mfma(vc[f % 3], pb[rg][ps], O[dt][rg]);
        if (f + 2 < kFrags) vc[(f + 2) % 3] = vop(vr[(f + 2) % (kPvAhead + 1)]);
      } else {
        const bf16x8_t v = vop(vr[f % (kPvAhead + 1)]);
#pragma unroll
        for (int rg = 0; rg < RG; ++rg) O[dt][rg] = mfma(v, pb[rg][ps], O[dt][rg]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int rg = 0; rg < RG; ++rg) l_run[rg] += psum[rg];
  }

  // ---- epilogue: normalise and write each row (out = O / l, lse = m + ln l).
  // The accumulator layout gives lane (n16, g) 16-byte chunk 4 dt + g of row
  // n16 for every column tile dt: fp32 rows are stored straight from there
  // (64-byte runs per row and instruction, which the L2 joins into whole
  // lines; measured faster than transposing through LDS first).  Splits of a
  // workspace of a megabyte or more write their rows as fp16 values divided
  // by the row's largest magnitude (kept in fp32 beside the lse): half the
  // bytes of fp32, at 2^-11 of that magnitude, which the combine multiplies
  // back; those
  // rows are transposed through LDS (a 32 KiB area per wave, 16-byte chunk c
  // of row rr in slot c ^ rr) and stored as contiguous 1 KiB rows.
  const bool direct = p.n_splits == 1;
  const bool half = !direct && p.ws_f16;
  const int64_t part = (int64_t)r * p.n_splits + s_idx;
  lds_barrier();  // every wave is done with the last block's LDS
  LDS uint8_t* const stage = smem + wave * 32768;
  const int ln = lds_opaque(lane);
#pragma unroll
  for (int rg = 0; rg < RG; ++rg) {
    const float l_tot = xor_sum(l_run[rg]);
    const int row0 = row_wg0 + wave * 16 * RG + rg * 16;
    const int row = row0 + n16;
    const float lse = l_tot > 0.f ? (m_run[rg] + __log2f(l_tot)) * kLn2 : -INFINITY;
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    if (!half) {
      if (g == 0 && row < p.rows) {
        if (direct) {
          const int i = row / p.H, hd = row - (row / p.H) * p.H;
          const int64_t lo = r * p.lse_s0 + i * p.lse_s1 + hd * p.lse_s2;
          if (p.out_wire) {
            // (m, l): the largest score, and the denominator relative to it
            // (l_tot is relative to the running maximum, which is at most m)
            p.lse[lo] = l_tot > 0.f ? m_true[rg] * kLn2 : -INFINITY;
            p.lse[lo + 1] = l_tot > 0.f ? l_tot * __builtin_amdgcn_exp2f(m_run[rg] - m_true[rg]) : 0.f;
          } else {
            p.lse[lo] = lse;
          }
        } else {
          p.ws_lse[part * p.rows + row] = lse;
          if (p.out_wire) p.ws_max[part * p.rows + row] = m_true[rg];
        }
      }
      if (row < p.rows && direct && p.out_wire) {
        // bf16 rows: 8-byte runs per row and instruction
        const int i = row / p.H, hd = row - (row / p.H) * p.H;
        uint16_t* dst = p.out16 + r * p.out_s0 + i * p.out_s1 + hd * p.out_s2;
#pragma unroll
        for (int dt = 0; dt < 32; ++dt) {
          f32x4_t v = O[dt][rg];
          asm volatile("" : "+a"(v));  // read in place, no copy back
          *(u16x4_t*)(dst + 4 * (4 * dt + g)) = f32x4_bf16(v * inv);
        }
      } else if (row < p.rows) {
        float* dst;
        if (direct) {
          const int i = row / p.H, hd = row - (row / p.H) * p.H;
          dst = p.out + r * p.out_s0 + i * p.out_s1 + hd * p.out_s2;
        } else {
          dst = p.ws_o32 + (part * p.rows + row) * kDLat;
        }
#pragma unroll
        for (int dt = 0; dt < 32; ++dt) {
          f32x4_t v = O[dt][rg];
          asm volatile("" : "+a"(v));  // read in place, no copy back
          *(f32x4_t*)(dst + 4 * (4 * dt + g)) = v * inv;
        }
      }
      continue;
    }
    // scaled fp16 rows: the row's largest magnitude, then the rows through LDS
    float amax = 0.f;
#pragma unroll
    for (int dt = 0; dt < 32; ++dt) {
      f32x4_t v = O[dt][rg];
      asm volatile("" : "+a"(v));
      v *= inv;
      amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
      *(LDS f32x4_t*)(stage + n16 * 2048 + (((4 * dt + g) ^ n16) << 4)) = v;
    }
    amax = xor_max(amax);
    const float row_scale = amax > 0.f ? amax : 1.f;
    if (g == 0 && row < p.rows) {
      p.ws_lse[part * p.rows + row] = lse;
      p.ws_scale[part * p.rows + row] = row_scale;
      if (p.out_wire) p.ws_max[part * p.rows + row] = m_true[rg];
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes are done
    // lane ln stores 16-byte chunk ln of row rr's 1 KiB fp16 row: columns
    // 8 ln .. 8 ln + 7, i.e. fp32 chunks 2 ln and 2 ln + 1 of the stage
    const float inv_scale_own = 1.f / row_scale;
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) {
      const int rw = row0 + rr;
      if (rw >= p.rows) break;
      // lane rr holds row rr's scale; a constant lane index reads it into a
      // scalar register
      const float is = __builtin_bit_cast(
          float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, inv_scale_own), rr));
      const f32x4_t a = *(const LDS f32x4_t*)(stage + rr * 2048 + (((2 * ln) ^ rr) << 4));
      const f32x4_t b = *(const LDS f32x4_t*)(stage + rr * 2048 + (((2 * ln + 1) ^ rr) << 4));
      u32x4_t h;
      h[0] = pack_f16(a[0] * is, a[1] * is);
      h[1] = pack_f16(a[2] * is, a[3] * is);
      h[2] = pack_f16(b[0] * is, b[1] * is);
      h[3] = pack_f16(b[2] * is, b[3] * is);
      *(u32x4_t*)(p.ws_o16 + (part * p.rows + rw) * kDLat + 8 * ln) = h;
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // reads of this row group done before it is overwritten
  }
}

}  // namespace

template <int KV, int SEL = kSelShared>
static void launch_kv(const PartialParams& p, int grid, int row_groups, hipStream_t s) {
  if (row_groups == 2)
    hipLaunchKernelGGL((partial_kernel<2, KV, SEL>), dim3(grid), dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL((partial_kernel<1, KV, SEL>), dim3(grid), dim3(256), 0, s, p);
}

hipError_t launch_partial(const PartialParams& p, int R, int kv, int row_groups, int sel_kind,
                          hipStream_t s) {
  const int grid = R * p.row_tiles * p.n_splits;
  if (grid <= 0) return hipSuccess;
  if (sel_kind == kSelPerRow) {
    if (kv == kKvFp8Shared)
      launch_kv<kKvFp8Shared, kSelPerRow>(p, grid, row_groups, s);
    else if (kv == kKvFp8Split)
      launch_kv<kKvFp8Split, kSelPerRow>(p, grid, row_groups, s);
    else
      launch_kv<kKvBf16, kSelPerRow>(p, grid, row_groups, s);
  } else if (sel_kind == kSelTokens) {
    if (kv == kKvFp8Shared)
      launch_kv<kKvFp8Shared, kSelTokens>(p, grid, row_groups, s);
    else if (kv == kKvFp8Split)
      launch_kv<kKvFp8Split, kSelTokens>(p, grid, row_groups, s);
    else
      launch_kv<kKvBf16, kSelTokens>(p, grid, row_groups, s);
  } else if (kv == kKvFp8Shared)
    launch_kv<kKvFp8Shared>(p, grid, row_groups, s);
  else if (kv == kKvFp8Split)
    launch_kv<kKvFp8Split>(p, grid, row_groups, s);
  else
    launch_kv<kKvBf16>(p, grid, row_groups, s);
  return hipGetLastError();
}

}  // namespace mla
