// Internal interface between the C-ABI host code and the HIP kernels of
// libmla_sparse.so.  Not installed; the public interface is mla_sparse.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mla {

constexpr int kDLat = 512;   // latent width (d_v)
constexpr int kDPe = 64;     // decoupled-RoPE width
constexpr int kBlock = 64;   // tokens per cache block
constexpr int kThreads = 256;             // merge / combine workgroup size
constexpr int kMaxSlotsPerSplit = 1024;   // selected-slot range one workgroup handles
constexpr int kMaxParts = 64;
// split-K workspaces of at least this many fp32 row bytes store scaled fp16
// rows (below it, as for a handful of rows, the shorter fp32 epilogue pays)
constexpr int64_t kWsHalfMinBytes = 1ll << 20;

// Partial attention over one (job, row tile, slot range) per workgroup.
struct PartialParams {
  const uint16_t* q_lat;  // bf16 bits
  const uint16_t* q_pe;
  int64_t ql_s0, ql_s1, ql_s2;  // element strides over (job, Mq, H)
  int64_t qp_s0, qp_s1, qp_s2;
  const uint8_t* ckv;  // pool base, bytes: [P][64][512] bf16 or e4m3 codes
  const uint8_t* kpe;  // [P][64][64]
  const float* ckv_scale;  // [P] (fp8 only)
  const float* kpe_scale;
  const int32_t* table;
  int64_t table_s0;
  const int32_t* sel;
  int64_t sel_s0;
  int64_t sel_s1;  // stride over query rows i: 0 when one selection serves the whole job
  int64_t P;
  int32_t NB, K;
  int32_t Mq, H, rows;  // rows = Mq * H
  int32_t n_splits, slots_per_split, row_tiles;
  // per-row selections split by logical block instead of by slot range: split
  // s takes blocks s, s + n_splits, ... from all K slots of every row
  int32_t split_by_id;
  // q rows shared by jobs: job r reads q row r % q_jobs; with q_rep =
  // jobs / q_jobs > 1 the work items of one q row's jobs are numbered next to
  // each other (so that they run on one XCD and read that row from one L2)
  int32_t q_jobs, q_rep;
  // work items numbered row tiles fastest (per-row selections split by
  // logical block, with enough row tiles that one split's tiles fill an XCD)
  int32_t tiles_fast;
  float scale_log2;  // softmax scale * log2(e)
  // destination: direct (n_splits == 1) or split-K workspace.  out_wire: the
  // bf16 wire form (Section 3.2): bf16 rows at out16 (element strides out_s*)
  // and (m, l) pairs at lse (pair strides lse_s*, in floats); else fp32 rows
  // at out and the lse at lse.
  int32_t out_wire;
  float* out;
  uint16_t* out16;
  int64_t out_s0, out_s1, out_s2;
  float* lse;
  int64_t lse_s0, lse_s1, lse_s2;
  // split-K workspace, [R][S][rows] split rows with their lse: fp32 rows, or
  // when ws_f16 is set (a megabyte of fp32 rows or more) fp16 rows divided
  // by the row's largest magnitude, which ws_scale holds
  int32_t ws_f16;
  float* ws_o32;     // [R][S][rows][512]
  uint16_t* ws_o16;  // [R][S][rows][512] fp16 bits
  float* ws_scale;   // [R][S][rows]
  float* ws_lse;     // [R][S][rows]
  float* ws_max;     // [R][S][rows], the split's largest score (log2 units; wire form)
};

// Combine of the S split partials of every job into the caller's outputs.
struct CombineParams {
  int32_t ws_f16;  // see PartialParams
  const float* ws_o32;
  const uint16_t* ws_o16;
  const float* ws_scale;
  const float* ws_lse;
  const float* ws_max;  // the splits' largest scores (log2 units), wire form only
  int32_t R, S, Mq, H, rows;
  int32_t out_wire;     // see PartialParams
  float* out;
  uint16_t* out16;
  int64_t out_s0, out_s1, out_s2;
  float* lse;
  int64_t lse_s0, lse_s1, lse_s2;
};

// Merge of n parts given by pointers with shared strides.  wire: the parts
// are in the bf16 wire form (bf16 rows, (m, l) pairs at lse[j] with strides
// l_s* in floats); else fp32 rows and lse values.
struct MergeParams {
  const void* o[kMaxParts];
  const float* lse[kMaxParts];
  int32_t wire;
  int32_t n_parts;
  int32_t B, Mq, H;
  int64_t o_s0, o_s1, o_s2;
  int64_t l_s0, l_s1, l_s2;
  float* out;
  int64_t out_s0, out_s1, out_s2;
  float* out_lse;  // may be null
  int64_t ol_s0, ol_s1, ol_s2;
};

// FETCH-side copy kernels: one workgroup moves 64 tokens of one layer.
struct FetchParams {
  // splice: chunk rows [L][n][D] -> pool rows; gather: pool rows -> out rows [L][K][D]
  const uint16_t* src_ckv;
  const uint16_t* src_kpe;
  uint16_t* dst_ckv;
  uint16_t* dst_kpe;
  const int32_t* table;  // logical block -> pool block
  const int32_t* sel;    // gather: selected logical tokens [K], -1 = empty
  int64_t P;             // pool blocks per layer
  int64_t n;             // tokens per layer: chunk tokens (splice) or slots K (gather)
  int64_t n_ids;         // gather: 64 * NB (logical tokens of the chunk)
  int64_t dst_start;     // splice: position of the chunk's first token in the requester's sequence
  int32_t L;
  int32_t pairing;       // 0: dims (2i, 2i+1); 1: dims (i, i + 32)
  float cs[32], sn[32];  // splice: cos, sin of delta * theta_i
};

hipError_t launch_fetch_gather(const FetchParams& p, hipStream_t s);
hipError_t launch_fetch_splice(const FetchParams& p, hipStream_t s);

// Cache kinds of the partial kernel.
constexpr int kKvBf16 = 0;
constexpr int kKvFp8Shared = 1;  // e4m3, one scale per block for ckv and kpe
constexpr int kKvFp8Split = 2;   // e4m3, separate ckv and kpe scales per block

// Per-row selections: the LDS counters of one workgroup's compaction live in
// its stage area, NB * (query rows of the tile) 16-bit counters.
constexpr int kPerRowCounterBytes = 2 * 64 * 1152 - 64;  // the stage area, less the wave counters
constexpr int kPerRowMaxRows = 64;                  // query rows per row tile (mask bits)
constexpr int kPerRowListFp8 = kMaxSlotsPerSplit / 2;  // list entries per split, fp8 caches

// Selection kinds: one block selection per job, one per query row, or one
// token selection per job (bf16 caches only for the last two).
constexpr int kSelShared = 0;
constexpr int kSelPerRow = 1;
constexpr int kSelTokens = 2;

// Launchers; return hipSuccess or the launch error.
// row_groups: 2 (row tiles of 128 rows) or 1 (row tiles of 64 rows)
hipError_t launch_partial(const PartialParams& p, int R, int kv, int row_groups, int sel_kind,
                          hipStream_t s);
hipError_t launch_combine(const CombineParams& p, hipStream_t s);
hipError_t launch_merge(const MergeParams& p, hipStream_t s);

}  // namespace mla
