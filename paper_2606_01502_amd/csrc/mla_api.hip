// C ABI of libmla_sparse.so: argument validation, the split-K plan, the
// split-K workspace and the kernel launches.  Declared in include/mla_sparse.h.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdint>
#include <map>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "../../include/mla_sparse.h"
#include "mla_kernels.h"

namespace {

thread_local std::string g_last_error;

mla_status_t fail(mla_status_t st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

struct Extent {
  uintptr_t lo, hi;  // [lo, hi) bytes touched
};

int dtype_size(int32_t dt) {
  switch (dt) {
    case MLA_DTYPE_BF16: return 2;
    case MLA_DTYPE_FP8_E4M3FN: return 1;
    case MLA_DTYPE_FP32: return 4;
    case MLA_DTYPE_INT32: return 4;
    default: return 0;
  }
}

int64_t numel(const mla_tensor_t& t) {
  int64_t n = 1;
  for (int d = 0; d < t.ndim; ++d) n *= t.shape[d];
  return n;
}

Extent extent(const mla_tensor_t& t) {
  const int es = dtype_size(t.dtype);
  if (numel(t) == 0) return {0, 0};
  int64_t hi = 0;
  for (int d = 0; d < t.ndim; ++d) hi += (t.shape[d] - 1) * t.stride[d];
  const uintptr_t base = reinterpret_cast<uintptr_t>(t.data);
  return {base, base + (uintptr_t)((hi + 1) * es)};
}

bool overlaps(const Extent& a, const Extent& b) {
  if (a.lo == a.hi || b.lo == b.hi) return false;
  return a.lo < b.hi && b.lo < a.hi;
}

// Common checks of one descriptor.  `name` is used in messages.
mla_status_t check_tensor(const mla_tensor_t* t, const char* name, int32_t dtype, int ndim,
                          bool allow_scale = false) {
  if (!t) return fail(MLA_ERR_INVALID_ARGUMENT, std::string(name) + ": null descriptor");
  if (t->dtype != dtype)
    return fail(MLA_ERR_INVALID_ARGUMENT, std::string(name) + ": wrong dtype " + std::to_string(t->dtype));
  if (t->ndim != ndim)
    return fail(MLA_ERR_INVALID_ARGUMENT, std::string(name) + ": expected " + std::to_string(ndim) +
                                              " dims, got " + std::to_string(t->ndim));
  for (int d = 0; d < ndim; ++d)
    if (t->shape[d] < 0 || t->stride[d] < 0)
      return fail(MLA_ERR_INVALID_ARGUMENT, std::string(name) + ": negative shape or stride");
  if (ndim > 0 && t->shape[ndim - 1] > 1 && t->stride[ndim - 1] != 1)
    return fail(MLA_ERR_INVALID_ARGUMENT, std::string(name) + ": innermost stride must be 1");
  if (numel(*t) > 0 && !t->data)
    return fail(MLA_ERR_INVALID_ARGUMENT, std::string(name) + ": null data pointer");
  if (!allow_scale && t->block_scale)
    return fail(MLA_ERR_INVALID_ARGUMENT, std::string(name) + ": block_scale must be NULL");
  return MLA_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Row-major contiguous with the given shape.
bool contiguous(const mla_tensor_t& t, std::initializer_list<int64_t> shape) {
  if (t.ndim != (int)shape.size()) return false;
  int d = 0;
  for (int64_t v : shape)
    if (t.shape[d++] != v) return false;
  int64_t st = 1;
  for (int k = t.ndim - 1; k >= 0; --k) {
    if (t.shape[k] > 1 && t.stride[k] != st) return false;
    st *= t.shape[k];
  }
  return true;
}

// Rows of a [.., .., .., D] tensor are 16-byte aligned: base and every outer stride.
bool rows_aligned(const mla_tensor_t& t, int es) {
  if (!aligned16(t.data)) return false;
  for (int d = 0; d + 1 < t.ndim; ++d)
    if ((t.stride[d] * es) % 16 != 0) return false;
  return true;
}

// Split-K workspace: one grow-only buffer per (device, stream).  The caller
// keeps `lock` (which holds g_ws_mutex) until both kernels that use the
// buffer are queued, so that calls from several host threads on one stream
// cannot queue a partial kernel between another call's partial and combine.
//
// A buffer is never freed while the process runs: a HIP graph captured on the
// stream keeps the address it was captured with, and replaying it after a
// larger call has replaced the buffer must still find that memory.  Replaced
// buffers are retired (kept), and each replacement at least doubles the size,
// so the retired ones together stay below the live one.  Growing is refused
// while the stream is being captured (an allocation there is not part of the
// graph, and under global capture it would invalidate the capture).
struct Workspace {
  void* ptr = nullptr;
  size_t bytes = 0;
};
std::mutex g_ws_mutex;
std::map<std::pair<int, hipStream_t>, Workspace> g_ws;
std::vector<void*> g_ws_retired;

mla_status_t get_workspace(hipStream_t stream, size_t bytes, void** out,
                           std::unique_lock<std::mutex>& lock) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(MLA_ERR_HIP, "hipGetDevice failed");
  lock = std::unique_lock<std::mutex>(g_ws_mutex);
  Workspace& ws = g_ws[{dev, stream}];
  if (ws.bytes < bytes) {
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(stream, &cap) != hipSuccess) {
      (void)hipGetLastError();
      return fail(MLA_ERR_HIP, "hipStreamIsCapturing failed");
    }
    if (cap != hipStreamCaptureStatusNone)
      return fail(MLA_ERR_UNSUPPORTED,
                  "the split-K workspace of this stream (" + std::to_string(ws.bytes) +
                      " bytes) is smaller than this call needs (" + std::to_string(bytes) +
                      ") and cannot grow during stream capture: make the call once on this "
                      "stream before capturing it");
    const size_t want = std::max({bytes, 2 * ws.bytes, (size_t)1 << 20});
    void* fresh = nullptr;
    if (hipMalloc(&fresh, want) != hipSuccess) {
      (void)hipGetLastError();
      return fail(MLA_ERR_OUT_OF_MEMORY, "split-K workspace allocation of " + std::to_string(want) + " bytes failed");
    }
    if (ws.ptr) g_ws_retired.push_back(ws.ptr);  // may still be in a captured graph
    ws.ptr = fresh;
    ws.bytes = want;
  }
  *out = ws.ptr;
  return MLA_OK;
}

// The split-K workspace of mla_sparse_partial_attn_noalloc: a static device
// array that the runtime places on every GPU the library runs on, held until
// the process ends.  Host code never uses its name as an address (on the host
// it names a stand-in); each device's address comes from hipGetSymbolAddress,
// taken once per device on the first call there, with that device current.
static __device__ __align__(256) uint8_t scratch[MLA_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

mla_status_t scratch_address(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(MLA_ERR_HIP, "hipGetDevice failed");
  if (dev < 0 || dev >= kMaxDevices) return fail(MLA_ERR_UNSUPPORTED, "device index beyond 64");
  std::lock_guard<std::mutex> guard(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      (void)hipGetLastError();
      return fail(MLA_ERR_HIP, std::string("hipGetSymbolAddress of the scratch array: ") +
                                   hipGetErrorString(e));
    }
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return MLA_OK;
}

int device_cus() {
  static int cus = 0;
  if (cus == 0) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
      cus = n;
    else
      cus = 256;
  }
  return cus;
}

// The partial call; `tokens`: sel names single logical tokens (block * 64 +
// t) rather than blocks; `no_alloc`: the split-K workspace is the static
// scratch array (nothing is allocated; sizes beyond it are refused).
mla_status_t partial_call(const mla_tensor_t* q_lat, const mla_tensor_t* q_pe,
                          const mla_tensor_t* ckv_pool, const mla_tensor_t* kpe_pool,
                          const mla_tensor_t* chunk_block_table,
                          const mla_tensor_t* sel_block_ids, float scale,
                          const mla_tensor_t* out_lat, const mla_tensor_t* out_lse,
                          const mla_partial_opts_t* opts, void* stream, bool tokens,
                          bool no_alloc = false) {
  try {
    g_last_error.clear();
    mla_status_t st;
    if ((st = check_tensor(q_lat, "q_lat", MLA_DTYPE_BF16, 4)) != MLA_OK) return st;
    if ((st = check_tensor(q_pe, "q_pe", MLA_DTYPE_BF16, 4)) != MLA_OK) return st;
    if (!ckv_pool || !kpe_pool) return fail(MLA_ERR_INVALID_ARGUMENT, "ckv_pool/kpe_pool: null descriptor");
    const int32_t kv_dtype = ckv_pool->dtype;
    if (kv_dtype != MLA_DTYPE_BF16 && kv_dtype != MLA_DTYPE_FP8_E4M3FN)
      return fail(MLA_ERR_INVALID_ARGUMENT, "ckv_pool: dtype must be bf16 or fp8-e4m3fn");
    const bool fp8 = kv_dtype == MLA_DTYPE_FP8_E4M3FN;
    if ((st = check_tensor(ckv_pool, "ckv_pool", kv_dtype, 3, fp8)) != MLA_OK) return st;
    if ((st = check_tensor(kpe_pool, "kpe_pool", kv_dtype, 3, fp8)) != MLA_OK) return st;
    if (fp8 && (!ckv_pool->block_scale || !kpe_pool->block_scale))
      return fail(MLA_ERR_INVALID_ARGUMENT, "fp8 pools need block_scale");
    if ((st = check_tensor(chunk_block_table, "chunk_block_table", MLA_DTYPE_INT32, 2)) != MLA_OK) return st;
    const bool per_row = !tokens && sel_block_ids && sel_block_ids->ndim == 3;
    const char* sel_name = tokens ? "sel_token_ids" : "sel_block_ids";
    if ((st = check_tensor(sel_block_ids, sel_name, MLA_DTYPE_INT32, per_row ? 3 : 2)) != MLA_OK)
      return st;
    const bool wire = opts && opts->out_format == MLA_OUT_BF16_WIRE;
    if ((st = check_tensor(out_lat, "out_lat", wire ? MLA_DTYPE_BF16 : MLA_DTYPE_FP32, 4)) != MLA_OK)
      return st;
    if ((st = check_tensor(out_lse, "out_lse", MLA_DTYPE_FP32, wire ? 4 : 3)) != MLA_OK) return st;
    if (opts) {
      for (int i = 0; i < 5; ++i)
        if (opts->reserved[i]) return fail(MLA_ERR_INVALID_ARGUMENT, "opts.reserved must be zero");
      if (opts->out_format != MLA_OUT_FP32 && opts->out_format != MLA_OUT_BF16_WIRE)
        return fail(MLA_ERR_INVALID_ARGUMENT, "opts.out_format must be MLA_OUT_FP32 or MLA_OUT_BF16_WIRE");
      if (opts->n_splits < 0) return fail(MLA_ERR_INVALID_ARGUMENT, "opts.n_splits must be >= 0");
      if (opts->row_tile != 0 && opts->row_tile != 64 && opts->row_tile != 128)
        return fail(MLA_ERR_INVALID_ARGUMENT, "opts.row_tile must be 0, 64 or 128");
    }

    // jobs come from the block table; q may hold fewer rows, R_q dividing R,
    // job r reading q row r mod R_q (one request's q shared by its chunks)
    const int64_t R = chunk_block_table->shape[0];
    const int64_t Rq = q_lat->shape[0], Mq = q_lat->shape[1], H = q_lat->shape[2];
    const int64_t P = ckv_pool->shape[0];
    const int64_t NB = chunk_block_table->shape[1], K = sel_block_ids->shape[per_row ? 2 : 1];
    auto shape_is = [](const mla_tensor_t* t, std::initializer_list<int64_t> s) {
      int d = 0;
      for (int64_t v : s)
        if (t->shape[d++] != v) return false;
      return true;
    };
    if (q_lat->shape[3] != MLA_DLAT) return fail(MLA_ERR_INVALID_ARGUMENT, "q_lat: last dim must be 512");
    if (R > 0 ? (Rq < 1 || R % Rq != 0) : Rq != 0)
      return fail(MLA_ERR_INVALID_ARGUMENT,
                  "q_lat: its first dim R_q must divide the number of jobs R (job r reads q row r mod R_q)");
    if (!shape_is(q_pe, {Rq, Mq, H, MLA_DPE})) return fail(MLA_ERR_INVALID_ARGUMENT, "q_pe: shape must be [R_q, Mq, H, 64]");
    if (!shape_is(ckv_pool, {P, MLA_BLOCK, MLA_DLAT})) return fail(MLA_ERR_INVALID_ARGUMENT, "ckv_pool: shape must be [P, 64, 512]");
    if (!shape_is(kpe_pool, {P, MLA_BLOCK, MLA_DPE})) return fail(MLA_ERR_INVALID_ARGUMENT, "kpe_pool: shape must be [P, 64, 64] with the P of ckv_pool");
    if (chunk_block_table->shape[0] != R) return fail(MLA_ERR_INVALID_ARGUMENT, "chunk_block_table: shape must be [R, NB]");
    if (sel_block_ids->shape[0] != R || (per_row && sel_block_ids->shape[1] != Mq))
      return fail(MLA_ERR_INVALID_ARGUMENT, "sel_block_ids: shape must be [R, K] or [R, Mq, K]");
    if (!shape_is(out_lat, {R, Mq, H, MLA_DLAT})) return fail(MLA_ERR_INVALID_ARGUMENT, "out_lat: shape must be [R, Mq, H, 512]");
    if (!wire && !shape_is(out_lse, {R, Mq, H}))
      return fail(MLA_ERR_INVALID_ARGUMENT, "out_lse: shape must be [R, Mq, H]");
    if (wire && (!shape_is(out_lse, {R, Mq, H, 2}) || out_lse->stride[3] != 1))
      return fail(MLA_ERR_INVALID_ARGUMENT, "out_lse: the wire form takes [R, Mq, H, 2] (m, l) pairs");
    if (ckv_pool->stride[0] != MLA_BLOCK * MLA_DLAT || ckv_pool->stride[1] != MLA_DLAT ||
        kpe_pool->stride[0] != MLA_BLOCK * MLA_DPE || kpe_pool->stride[1] != MLA_DPE)
      return fail(MLA_ERR_INVALID_ARGUMENT, "pools must be contiguous");
    if (!aligned16(ckv_pool->data) || !aligned16(kpe_pool->data))
      return fail(MLA_ERR_INVALID_ARGUMENT, "pools must be 16-byte aligned");
    if (!rows_aligned(*q_lat, 2) || !rows_aligned(*q_pe, 2))
      return fail(MLA_ERR_INVALID_ARGUMENT, "q_lat/q_pe rows must be 16-byte aligned");
    if (!rows_aligned(*out_lat, wire ? 2 : 4))
      return fail(MLA_ERR_INVALID_ARGUMENT, "out_lat rows must be 16-byte aligned");
    if (wire && ((reinterpret_cast<uintptr_t>(out_lse->data) & 7u) != 0 || out_lse->stride[0] % 2 ||
                 out_lse->stride[1] % 2 || out_lse->stride[2] % 2))
      return fail(MLA_ERR_INVALID_ARGUMENT, "out_lse (m, l) pairs must be 8-byte aligned");
    // |scale| <= 2^64 keeps scale * log2(e) and the scores of any bf16 or fp8
    // rows whose dot products stay below 2^63 finite in fp32
    if (!(std::fabs(scale) <= 18446744073709551616.0f))
      return fail(MLA_ERR_INVALID_ARGUMENT, "scale must be finite with |scale| <= 2^64");
    if (R > INT32_MAX || Mq * H > (1 << 24) || K > INT32_MAX || NB > INT32_MAX || P > INT32_MAX)
      return fail(MLA_ERR_UNSUPPORTED, "sizes beyond the int32 index range");
    if (tokens && (NB > (INT32_MAX >> 6) || P > (INT32_MAX >> 6)))
      return fail(MLA_ERR_UNSUPPORTED, "token selections: NB or P beyond 2^25 blocks");

    const Extent outs[2] = {extent(*out_lat), extent(*out_lse)};
    auto scale_extent = [&](const float* sc) -> Extent {
      if (!fp8 || P == 0) return {0, 0};
      return {(uintptr_t)sc, (uintptr_t)(sc + P)};
    };
    const Extent ins[8] = {extent(*q_lat), extent(*q_pe), extent(*ckv_pool), extent(*kpe_pool),
                           extent(*chunk_block_table), extent(*sel_block_ids),
                           scale_extent(ckv_pool->block_scale), scale_extent(kpe_pool->block_scale)};
    if (overlaps(outs[0], outs[1])) return fail(MLA_ERR_INVALID_ARGUMENT, "out_lat and out_lse overlap");
    for (const Extent& o : outs)
      for (const Extent& i : ins)
        if (overlaps(o, i)) return fail(MLA_ERR_INVALID_ARGUMENT, "an output overlaps an input");

    const int64_t rows = Mq * H;
    if (R == 0 || rows == 0) return MLA_OK;

    // ---- plan: row tiles of 128 or 64 rows (4 waves of 32 or 16 rows);
    // split-K over slot ranges so that the grid covers the chip
    // slots in 64-token blocks (a token selection's slots fill K / 64 blocks)
    const int64_t Kb = tokens ? (K + 63) / 64 : K;
    int row_groups = rows > 64 ? 2 : 1;
    if (opts && opts->row_tile) {
      row_groups = opts->row_tile / 64;
    } else if (row_groups == 2) {
      // 128-row tiles read each block once for twice the rows, which pays
      // when splits are long; when the grid covers the chip only with short
      // splits (under 8 blocks each), 64-row tiles finish sooner: twice the
      // work items, each with half the fixed cost (query rows in, partial
      // rows out)
      const int64_t units2 = R * ((rows + 127) / 128);
      const int64_t s2 = std::min<int64_t>((device_cus() + units2 - 1) / units2,
                                           std::max<int64_t>(Kb / 2, 1));
      if (Kb < 8 * s2) row_groups = 1;
    }
    // per-row selections: the query rows a row tile spans (one mask bit each)
    auto tile_query_rows = [&](int rg) {
      const int64_t rw = 64 * rg;
      int64_t most = 0;
      for (int64_t r0 = 0; r0 < rows; r0 += rw) {
        const int64_t last = std::min<int64_t>(r0 + rw, rows) - 1;
        most = std::max<int64_t>(most, last / H - r0 / H + 1);
      }
      return most;
    };
    int64_t tile_qrows = 1;
    if (per_row) {
      if (row_groups == 2 && tile_query_rows(2) > mla::kPerRowMaxRows) {
        if (opts && opts->row_tile == 128)
          return fail(MLA_ERR_UNSUPPORTED, "per-row selections: too many query rows per 128-row tile");
        row_groups = 1;
      }
      tile_qrows = tile_query_rows(row_groups);
      if (tile_qrows > mla::kPerRowMaxRows)
        return fail(MLA_ERR_UNSUPPORTED, "per-row selections: too many query rows per tile");
      if (NB * tile_qrows * 2 > mla::kPerRowCounterBytes)
        return fail(MLA_ERR_UNSUPPORTED, "per-row selections: NB x query rows per tile too large");
    }
    const int rows_wg = 64 * row_groups;
    const int64_t row_tiles = (rows + rows_wg - 1) / rows_wg;
    // per-row selections whose tile slots all fit one list split by logical
    // block: every split then scans all slots and the rows that chose a block
    // in different slots still share its load
    // entries one split's list holds (per-row selections with an fp8 cache:
    // half a list, see the kernel's LDS layout)
    const int64_t list_cap = per_row && fp8 ? mla::kPerRowListFp8 : mla::kMaxSlotsPerSplit;
    const bool by_id = per_row && tile_qrows > 1 && K * tile_qrows <= list_cap;
    int64_t S;
    if (opts && opts->n_splits > 0) {
      S = std::min<int64_t>(opts->n_splits, std::max<int64_t>(by_id ? NB : K, 1));
    } else if (by_id) {
      const int64_t units = R * row_tiles;
      S = std::max<int64_t>(1, (device_cus() + units - 1) / units);
      S = std::min<int64_t>(S, std::max<int64_t>(std::min<int64_t>(NB, K * tile_qrows) / 2, 1));
    } else {
      // enough work items to cover the chip, but at least two slots per split:
      // a split of one block costs more in fixed latency (its prologue,
      // epilogue and share of the combine) than the block itself
      const int64_t units = R * row_tiles;
      S = std::max<int64_t>(1, (device_cus() + units - 1) / units);
      S = std::min<int64_t>(S, std::max<int64_t>(Kb / 2, 1));
      // two splits of at most two blocks save at most two blocks' time and
      // add the combine's launch: one split does better (4 blocks of one
      // 16-row job: 12.4 us in one split against 14.9 in two)
      if (S == 2 && Kb <= 5) S = 1;
    }
    // a split's block list holds at most kMaxSlotsPerSplit entries: its slots,
    // or for per-row selections its slots of every query row of the tile
    int64_t sps = K;
    if (tokens) {
      // whole virtual blocks per split, at most one list of tokens
      S = std::max<int64_t>(S, (K + mla::kMaxSlotsPerSplit - 1) / mla::kMaxSlotsPerSplit);
      sps = std::max<int64_t>(64, ((K + S - 1) / S + 63) / 64 * 64);
      sps = std::min<int64_t>(sps, mla::kMaxSlotsPerSplit);
      S = std::max<int64_t>(1, (K + sps - 1) / sps);
    } else if (!by_id) {
      S = std::max<int64_t>(S, (K * tile_qrows + list_cap - 1) / list_cap);
      sps = std::max<int64_t>(1, (K + S - 1) / S);
      if (per_row) sps = std::min<int64_t>(sps, std::max<int64_t>(1, list_cap / tile_qrows));
      S = std::max<int64_t>(1, (K + sps - 1) / sps);
    }
    if (R * row_tiles * S > INT32_MAX) return fail(MLA_ERR_UNSUPPORTED, "grid too large");

    hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
    mla::PartialParams p{};
    p.q_lat = (const uint16_t*)q_lat->data;
    p.q_pe = (const uint16_t*)q_pe->data;
    p.ql_s0 = q_lat->stride[0]; p.ql_s1 = q_lat->stride[1]; p.ql_s2 = q_lat->stride[2];
    p.qp_s0 = q_pe->stride[0]; p.qp_s1 = q_pe->stride[1]; p.qp_s2 = q_pe->stride[2];
    p.ckv = (const uint8_t*)ckv_pool->data;
    p.kpe = (const uint8_t*)kpe_pool->data;
    p.ckv_scale = ckv_pool->block_scale;
    p.kpe_scale = kpe_pool->block_scale;
    p.table = (const int32_t*)chunk_block_table->data;
    p.table_s0 = chunk_block_table->stride[0];
    p.sel = (const int32_t*)sel_block_ids->data;
    p.sel_s0 = sel_block_ids->stride[0];
    p.sel_s1 = per_row ? sel_block_ids->stride[1] : 0;
    p.P = P;
    p.NB = (int32_t)NB;
    p.K = (int32_t)K;
    p.Mq = (int32_t)Mq;
    p.H = (int32_t)H;
    p.rows = (int32_t)rows;
    p.n_splits = (int32_t)S;
    p.slots_per_split = (int32_t)sps;
    p.split_by_id = by_id ? 1 : 0;
    p.q_jobs = (int32_t)std::max<int64_t>(Rq, 1);
    p.q_rep = (int32_t)(Rq > 0 ? R / Rq : 1);
    // split-major numbering once a split's row tiles fill an XCD's share of
    // the grid (below that the combine's reads of a tile's splits on one XCD
    // are worth more than the shared block loads)
    p.tiles_fast = by_id && row_tiles >= 8 ? 1 : 0;
    p.row_tiles = (int32_t)row_tiles;
    p.scale_log2 = (float)((double)scale * 1.4426950408889634074);
    p.out_wire = wire ? 1 : 0;
    p.out16 = (uint16_t*)out_lat->data;
    p.out = (float*)out_lat->data;
    p.out_s0 = out_lat->stride[0]; p.out_s1 = out_lat->stride[1]; p.out_s2 = out_lat->stride[2];
    p.lse = (float*)out_lse->data;
    p.lse_s0 = out_lse->stride[0]; p.lse_s1 = out_lse->stride[1]; p.lse_s2 = out_lse->stride[2];
    std::unique_lock<std::mutex> ws_lock;  // held until the combine is queued
    if (S > 1) {
      // split rows, then their scales (fp16 rows only), then their lse values.
      // fp16 rows halve the workspace round trip, which pays from about a
      // megabyte of split rows on; tiny workspaces keep fp32 rows, whose
      // epilogue is a little shorter
      const size_t n_part_rows = (size_t)R * S * rows;
      p.ws_f16 = n_part_rows * MLA_DLAT * sizeof(float) >= (size_t)mla::kWsHalfMinBytes;
      const size_t o_bytes = n_part_rows * MLA_DLAT * (p.ws_f16 ? sizeof(uint16_t) : sizeof(float));
      const size_t ws_bytes = o_bytes + 3 * n_part_rows * sizeof(float);
      void* ws = nullptr;
      if (no_alloc) {
        if (ws_bytes > (size_t)MLA_NOALLOC_SCRATCH_BYTES)
          return fail(MLA_ERR_UNSUPPORTED,
                      "this call's split-K partials need " + std::to_string(ws_bytes) +
                          " bytes, more than the " + std::to_string((long long)MLA_NOALLOC_SCRATCH_BYTES) +
                          "-byte scratch array of the allocation-free entry point (fewer jobs or "
                          "splits per call)");
        if ((st = scratch_address(&ws)) != MLA_OK) return st;
      } else if ((st = get_workspace(hs, ws_bytes, &ws, ws_lock)) != MLA_OK) {
        return st;
      }
      p.ws_o32 = (float*)ws;
      p.ws_o16 = (uint16_t*)ws;
      p.ws_scale = (float*)((char*)ws + o_bytes);
      p.ws_lse = p.ws_scale + n_part_rows;
      p.ws_max = p.ws_lse + n_part_rows;
    }
    const int kv = !fp8 ? mla::kKvBf16
                 : (ckv_pool->block_scale == kpe_pool->block_scale ? mla::kKvFp8Shared
                                                                   : mla::kKvFp8Split);
    const int sel_kind = tokens ? mla::kSelTokens : per_row ? mla::kSelPerRow : mla::kSelShared;
    hipError_t e = mla::launch_partial(p, (int)R, kv, row_groups, sel_kind, hs);
    if (e != hipSuccess) return fail(MLA_ERR_HIP, std::string("partial kernel launch: ") + hipGetErrorString(e));
    if (S > 1) {
      mla::CombineParams c{};
      c.ws_f16 = p.ws_f16;
      c.ws_o32 = p.ws_o32;
      c.ws_o16 = p.ws_o16;
      c.ws_scale = p.ws_scale;
      c.ws_lse = p.ws_lse;
      c.ws_max = p.ws_max;
      c.R = (int32_t)R; c.S = (int32_t)S; c.Mq = (int32_t)Mq; c.H = (int32_t)H; c.rows = (int32_t)rows;
      c.out_wire = p.out_wire;
      c.out16 = p.out16;
      c.out = p.out; c.out_s0 = p.out_s0; c.out_s1 = p.out_s1; c.out_s2 = p.out_s2;
      c.lse = p.lse; c.lse_s0 = p.lse_s0; c.lse_s1 = p.lse_s1; c.lse_s2 = p.lse_s2;
      e = mla::launch_combine(c, hs);
      if (e != hipSuccess) return fail(MLA_ERR_HIP, std::string("combine kernel launch: ") + hipGetErrorString(e));
    }
    return MLA_OK;
  } catch (...) {
    return fail(MLA_ERR_HIP, "internal error");
  }
}

}  // namespace

extern "C" {

const char* mla_last_error(void) { return g_last_error.c_str(); }

int32_t mla_version(void) { return MLA_SPARSE_VERSION; }

mla_status_t mla_sparse_partial_attn_ex(const mla_tensor_t* q_lat, const mla_tensor_t* q_pe,
                                        const mla_tensor_t* ckv_pool, const mla_tensor_t* kpe_pool,
                                        const mla_tensor_t* chunk_block_table,
                                        const mla_tensor_t* sel_block_ids, float scale,
                                        const mla_tensor_t* out_lat, const mla_tensor_t* out_lse,
                                        const mla_partial_opts_t* opts, void* stream) {
  return partial_call(q_lat, q_pe, ckv_pool, kpe_pool, chunk_block_table, sel_block_ids, scale,
                      out_lat, out_lse, opts, stream, false);
}

mla_status_t mla_sparse_partial_attn_noalloc(const mla_tensor_t* q_lat, const mla_tensor_t* q_pe,
                                             const mla_tensor_t* ckv_pool,
                                             const mla_tensor_t* kpe_pool,
                                             const mla_tensor_t* chunk_block_table,
                                             const mla_tensor_t* sel_block_ids, float scale,
                                             const mla_tensor_t* out_lat,
                                             const mla_tensor_t* out_lse,
                                             const mla_partial_opts_t* opts, void* stream) {
  return partial_call(q_lat, q_pe, ckv_pool, kpe_pool, chunk_block_table, sel_block_ids, scale,
                      out_lat, out_lse, opts, stream, false, true);
}

mla_status_t mla_sparse_partial_attn_tokens(const mla_tensor_t* q_lat, const mla_tensor_t* q_pe,
                                            const mla_tensor_t* ckv_pool,
                                            const mla_tensor_t* kpe_pool,
                                            const mla_tensor_t* chunk_block_table,
                                            const mla_tensor_t* sel_token_ids, float scale,
                                            const mla_tensor_t* out_lat,
                                            const mla_tensor_t* out_lse,
                                            const mla_partial_opts_t* opts, void* stream) {
  return partial_call(q_lat, q_pe, ckv_pool, kpe_pool, chunk_block_table, sel_token_ids, scale,
                      out_lat, out_lse, opts, stream, true);
}

mla_status_t mla_primitive_costs(const mla_cost_model_t* m, const mla_cost_case_t* c,
                                 mla_cost_t* out) {
  g_last_error.clear();
  if (!m || !c || !out) return fail(MLA_ERR_INVALID_ARGUMENT, "null pointer");
  const double consts[] = {m->probe_us, m->compute_us, m->merge_us, m->splice_us, m->prefill_us};
  for (double v : consts)
    if (!(v >= 0.0) || !std::isfinite(v))
      return fail(MLA_ERR_INVALID_ARGUMENT, "model times must be finite and >= 0");
  if (!(m->route_bw_gbs > 0.0) || !(m->pull_bw_gbs > 0.0) || !std::isfinite(m->route_bw_gbs) ||
      !std::isfinite(m->pull_bw_gbs))
    return fail(MLA_ERR_INVALID_ARGUMENT, "throughputs must be finite and > 0");
  if (m->layers < 1 || m->reserved) return fail(MLA_ERR_INVALID_ARGUMENT, "layers must be >= 1, reserved 0");
  if (c->mq < 0 || c->q_bytes < 0 || c->p_bytes < 0 || c->chunk_tokens < 1 || c->kv_bytes < 1)
    return fail(MLA_ERR_INVALID_ARGUMENT, "sizes: mq, q, p >= 0; chunk_tokens, kv_bytes >= 1");
  // bytes / (GB/s) = 1e-9 s per byte = 1e-3 us per byte
  const double row = (double)c->q_bytes + (double)c->p_bytes;  // q + p, one routed row
  const double routed = (double)c->mq * row;                    // Mq (q + p)
  const double layer_chunk = (double)c->chunk_tokens * (double)c->kv_bytes;  // c_t b_KV
  const double L = (double)m->layers;
  mla_cost_t r{};
  r.route_us = m->probe_us + routed / (m->route_bw_gbs * 1e3) + m->compute_us + m->merge_us;
  r.fetch_us = L * layer_chunk / (m->pull_bw_gbs * 1e3) + m->splice_us;
  r.local_us = (double)c->chunk_tokens * L * m->prefill_us;
  r.choice = MLA_PRIMITIVE_ROUTE;
  double best = r.route_us;
  if (r.fetch_us < best) { r.choice = MLA_PRIMITIVE_FETCH; best = r.fetch_us; }
  if (r.local_us < best) r.choice = MLA_PRIMITIVE_LOCAL;
  r.wire_crossover_mq = row > 0.0 ? layer_chunk / row : INFINITY;
  r.wire_saving = 1.0 - routed / layer_chunk;
  r.congestion_bw_gbs = m->splice_us > 0.0 ? routed / (m->splice_us * 1e3) : INFINITY;
  r.splice_crossover_tokens = m->prefill_us > 0.0 ? m->splice_us / (L * m->prefill_us) : INFINITY;
  *out = r;
  return MLA_OK;
}

mla_status_t mla_fetch_gather(const mla_tensor_t* ckv_pool, const mla_tensor_t* kpe_pool,
                              const mla_tensor_t* chunk_block_table,
                              const mla_tensor_t* sel_token_ids, const mla_tensor_t* out_ckv,
                              const mla_tensor_t* out_kpe, void* stream) {
  try {
    g_last_error.clear();
    mla_status_t st;
    if ((st = check_tensor(ckv_pool, "ckv_pool", MLA_DTYPE_BF16, 4)) != MLA_OK) return st;
    if ((st = check_tensor(kpe_pool, "kpe_pool", MLA_DTYPE_BF16, 4)) != MLA_OK) return st;
    if ((st = check_tensor(chunk_block_table, "chunk_block_table", MLA_DTYPE_INT32, 1)) != MLA_OK) return st;
    if ((st = check_tensor(sel_token_ids, "sel_token_ids", MLA_DTYPE_INT32, 1)) != MLA_OK) return st;
    if ((st = check_tensor(out_ckv, "out_ckv", MLA_DTYPE_BF16, 3)) != MLA_OK) return st;
    if ((st = check_tensor(out_kpe, "out_kpe", MLA_DTYPE_BF16, 3)) != MLA_OK) return st;
    const int64_t L = ckv_pool->shape[0], P = ckv_pool->shape[1];
    const int64_t NB = chunk_block_table->shape[0], K = sel_token_ids->shape[0];
    if (!contiguous(*ckv_pool, {L, P, MLA_BLOCK, MLA_DLAT}) || !contiguous(*kpe_pool, {L, P, MLA_BLOCK, MLA_DPE}))
      return fail(MLA_ERR_INVALID_ARGUMENT, "pools must be contiguous [L, P, 64, 512] and [L, P, 64, 64]");
    if (!contiguous(*chunk_block_table, {NB}) || !contiguous(*sel_token_ids, {K}))
      return fail(MLA_ERR_INVALID_ARGUMENT, "chunk_block_table and sel_token_ids must be contiguous");
    if (!contiguous(*out_ckv, {L, K, MLA_DLAT}) || !contiguous(*out_kpe, {L, K, MLA_DPE}))
      return fail(MLA_ERR_INVALID_ARGUMENT, "out_ckv / out_kpe must be contiguous [L, K, 512] / [L, K, 64]");
    if (!aligned16(ckv_pool->data) || !aligned16(kpe_pool->data) || !aligned16(out_ckv->data) ||
        !aligned16(out_kpe->data))
      return fail(MLA_ERR_INVALID_ARGUMENT, "pools and outputs must be 16-byte aligned");
    if (NB > (INT32_MAX >> 6) || P > INT32_MAX || L * ((K + 63) / 64) > INT32_MAX)
      return fail(MLA_ERR_UNSUPPORTED, "sizes beyond the index range");
    const Extent outs[2] = {extent(*out_ckv), extent(*out_kpe)};
    const Extent ins[4] = {extent(*ckv_pool), extent(*kpe_pool), extent(*chunk_block_table),
                           extent(*sel_token_ids)};
    if (overlaps(outs[0], outs[1])) return fail(MLA_ERR_INVALID_ARGUMENT, "out_ckv and out_kpe overlap");
    for (const Extent& o : outs)
      for (const Extent& i : ins)
        if (overlaps(o, i)) return fail(MLA_ERR_INVALID_ARGUMENT, "an output overlaps an input");
    mla::FetchParams p{};
    p.src_ckv = (const uint16_t*)ckv_pool->data;
    p.src_kpe = (const uint16_t*)kpe_pool->data;
    p.dst_ckv = (uint16_t*)out_ckv->data;
    p.dst_kpe = (uint16_t*)out_kpe->data;
    p.table = (const int32_t*)chunk_block_table->data;
    p.sel = (const int32_t*)sel_token_ids->data;
    p.P = P;
    p.n = K;
    p.n_ids = NB * MLA_BLOCK;
    p.L = (int32_t)L;
    hipError_t e = mla::launch_fetch_gather(p, reinterpret_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(MLA_ERR_HIP, std::string("gather kernel launch: ") + hipGetErrorString(e));
    return MLA_OK;
  } catch (...) {
    return fail(MLA_ERR_HIP, "internal error");
  }
}

mla_status_t mla_fetch_splice(const mla_tensor_t* chunk_ckv, const mla_tensor_t* chunk_kpe,
                              const mla_tensor_t* ckv_pool, const mla_tensor_t* kpe_pool,
                              const mla_tensor_t* block_table, int64_t dst_start, int64_t delta,
                              float rope_base, int32_t pairing, void* stream) {
  try {
    g_last_error.clear();
    mla_status_t st;
    if ((st = check_tensor(chunk_ckv, "chunk_ckv", MLA_DTYPE_BF16, 3)) != MLA_OK) return st;
    if ((st = check_tensor(chunk_kpe, "chunk_kpe", MLA_DTYPE_BF16, 3)) != MLA_OK) return st;
    if ((st = check_tensor(ckv_pool, "ckv_pool", MLA_DTYPE_BF16, 4)) != MLA_OK) return st;
    if ((st = check_tensor(kpe_pool, "kpe_pool", MLA_DTYPE_BF16, 4)) != MLA_OK) return st;
    if ((st = check_tensor(block_table, "block_table", MLA_DTYPE_INT32, 1)) != MLA_OK) return st;
    const int64_t L = chunk_ckv->shape[0], n = chunk_ckv->shape[1];
    const int64_t P = ckv_pool->shape[1], NB = block_table->shape[0];
    if (!contiguous(*chunk_ckv, {L, n, MLA_DLAT}) || !contiguous(*chunk_kpe, {L, n, MLA_DPE}))
      return fail(MLA_ERR_INVALID_ARGUMENT, "chunk_ckv / chunk_kpe must be contiguous [L, n, 512] / [L, n, 64]");
    if (!contiguous(*ckv_pool, {L, P, MLA_BLOCK, MLA_DLAT}) || !contiguous(*kpe_pool, {L, P, MLA_BLOCK, MLA_DPE}))
      return fail(MLA_ERR_INVALID_ARGUMENT, "pools must be contiguous [L, P, 64, 512] and [L, P, 64, 64] with the chunk's L");
    if (!contiguous(*block_table, {NB})) return fail(MLA_ERR_INVALID_ARGUMENT, "block_table must be contiguous");
    if (!aligned16(chunk_ckv->data) || !aligned16(chunk_kpe->data) || !aligned16(ckv_pool->data) ||
        !aligned16(kpe_pool->data))
      return fail(MLA_ERR_INVALID_ARGUMENT, "chunk and pools must be 16-byte aligned");
    if (pairing != 0 && pairing != 1) return fail(MLA_ERR_INVALID_ARGUMENT, "pairing must be 0 or 1");
    if (!(rope_base > 0.f) || !std::isfinite(rope_base))
      return fail(MLA_ERR_INVALID_ARGUMENT, "rope_base must be finite and > 0");
    if (dst_start < 0 || dst_start > NB * MLA_BLOCK - n)
      return fail(MLA_ERR_INVALID_ARGUMENT, "the chunk must fit the block table: 0 <= dst_start, dst_start + n <= 64 NB");
    if (P > INT32_MAX || L * ((n + 63) / 64) > INT32_MAX)
      return fail(MLA_ERR_UNSUPPORTED, "sizes beyond the index range");
    const Extent outs[2] = {extent(*ckv_pool), extent(*kpe_pool)};
    const Extent ins[3] = {extent(*chunk_ckv), extent(*chunk_kpe), extent(*block_table)};
    if (overlaps(outs[0], outs[1])) return fail(MLA_ERR_INVALID_ARGUMENT, "ckv_pool and kpe_pool overlap");
    for (const Extent& o : outs)
      for (const Extent& i : ins)
        if (overlaps(o, i)) return fail(MLA_ERR_INVALID_ARGUMENT, "a pool overlaps the chunk or the table");
    mla::FetchParams p{};
    p.src_ckv = (const uint16_t*)chunk_ckv->data;
    p.src_kpe = (const uint16_t*)chunk_kpe->data;
    p.dst_ckv = (uint16_t*)ckv_pool->data;
    p.dst_kpe = (uint16_t*)kpe_pool->data;
    p.table = (const int32_t*)block_table->data;
    p.P = P;
    p.n = n;
    p.dst_start = dst_start;
    p.L = (int32_t)L;
    p.pairing = pairing;
    // pair i turns through delta * base^(-2i/64), evaluated in double
    for (int i = 0; i < MLA_DPE / 2; ++i) {
      const double ang = (double)delta * std::pow((double)rope_base, -2.0 * i / MLA_DPE);
      p.cs[i] = (float)std::cos(ang);
      p.sn[i] = (float)std::sin(ang);
    }
    hipError_t e = mla::launch_fetch_splice(p, reinterpret_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(MLA_ERR_HIP, std::string("splice kernel launch: ") + hipGetErrorString(e));
    return MLA_OK;
  } catch (...) {
    return fail(MLA_ERR_HIP, "internal error");
  }
}

mla_status_t mla_sparse_partial_attn(const mla_tensor_t* q_lat, const mla_tensor_t* q_pe,
                                     const mla_tensor_t* ckv_pool, const mla_tensor_t* kpe_pool,
                                     const mla_tensor_t* chunk_block_table,
                                     const mla_tensor_t* sel_block_ids, float scale,
                                     const mla_tensor_t* out_lat, const mla_tensor_t* out_lse,
                                     void* stream) {
  return mla_sparse_partial_attn_ex(q_lat, q_pe, ckv_pool, kpe_pool, chunk_block_table,
                                    sel_block_ids, scale, out_lat, out_lse, nullptr, stream);
}

mla_status_t mla_merge_partials_ex(const mla_tensor_t* const* out_lat,
                                   const mla_tensor_t* const* out_lse, int32_t n_parts,
                                   const mla_tensor_t* out, const mla_tensor_t* merged_lse,
                                   void* stream) {
  try {
    g_last_error.clear();
    if (n_parts < 1 || n_parts > MLA_MAX_PARTS)
      return fail(MLA_ERR_INVALID_ARGUMENT, "n_parts must be in 1.." + std::to_string(MLA_MAX_PARTS));
    if (!out_lat || !out_lse) return fail(MLA_ERR_INVALID_ARGUMENT, "null part arrays");
    mla_status_t st;
    if ((st = check_tensor(out, "out", MLA_DTYPE_FP32, 4)) != MLA_OK) return st;
    if (out->shape[3] != MLA_DLAT) return fail(MLA_ERR_INVALID_ARGUMENT, "out: last dim must be 512");
    // parts in the bf16 wire form: bf16 rows with (m, l) pairs
    const bool wire = out_lat[0] && out_lat[0]->dtype == MLA_DTYPE_BF16;
    if (!rows_aligned(*out, 4)) return fail(MLA_ERR_INVALID_ARGUMENT, "out rows must be 16-byte aligned");
    if (merged_lse) {
      if ((st = check_tensor(merged_lse, "merged_lse", MLA_DTYPE_FP32, 3)) != MLA_OK) return st;
      for (int d = 0; d < 3; ++d)
        if (merged_lse->shape[d] != out->shape[d])
          return fail(MLA_ERR_INVALID_ARGUMENT, "merged_lse: shape must be [B, Mq, H]");
    }
    mla::MergeParams p{};
    std::string nm;
    for (int j = 0; j < n_parts; ++j) {
      nm = "out_lat[" + std::to_string(j) + "]";
      if ((st = check_tensor(out_lat[j], nm.c_str(), wire ? MLA_DTYPE_BF16 : MLA_DTYPE_FP32, 4)) != MLA_OK)
        return st;
      nm = "out_lse[" + std::to_string(j) + "]";
      if ((st = check_tensor(out_lse[j], nm.c_str(), MLA_DTYPE_FP32, wire ? 4 : 3)) != MLA_OK) return st;
      for (int d = 0; d < 4; ++d)
        if (out_lat[j]->shape[d] != out->shape[d])
          return fail(MLA_ERR_INVALID_ARGUMENT, "out_lat parts must have the shape of out");
      for (int d = 0; d < 3; ++d)
        if (out_lse[j]->shape[d] != out->shape[d])
          return fail(MLA_ERR_INVALID_ARGUMENT, "out_lse parts must be [B, Mq, H]");
      if (wire && (out_lse[j]->shape[3] != 2 || out_lse[j]->stride[3] != 1 ||
                   (reinterpret_cast<uintptr_t>(out_lse[j]->data) & 7u) != 0 ||
                   out_lse[j]->stride[0] % 2 || out_lse[j]->stride[1] % 2 || out_lse[j]->stride[2] % 2))
        return fail(MLA_ERR_INVALID_ARGUMENT,
                    "wire-form parts: out_lse must be [B, Mq, H, 2] fp32 (m, l) pairs, 8-byte aligned");
      for (int d = 0; d < 3; ++d)
        if (out_lat[j]->stride[d] != out_lat[0]->stride[d] || out_lse[j]->stride[d] != out_lse[0]->stride[d])
          return fail(MLA_ERR_UNSUPPORTED, "parts must share one set of strides");
      if (!rows_aligned(*out_lat[j], wire ? 2 : 4))
        return fail(MLA_ERR_INVALID_ARGUMENT, "part rows must be 16-byte aligned");
      const Extent eo = extent(*out);
      if (overlaps(eo, extent(*out_lat[j])) || overlaps(eo, extent(*out_lse[j])))
        return fail(MLA_ERR_INVALID_ARGUMENT, "out overlaps an input part");
      if (merged_lse) {
        const Extent el = extent(*merged_lse);
        if (overlaps(el, extent(*out_lat[j])) || overlaps(el, extent(*out_lse[j])) || overlaps(el, eo))
          return fail(MLA_ERR_INVALID_ARGUMENT, "merged_lse overlaps another tensor");
      }
      p.o[j] = out_lat[j]->data;
      p.lse[j] = (const float*)out_lse[j]->data;
    }
    const int64_t B = out->shape[0], Mq = out->shape[1], H = out->shape[2];
    if (B * Mq * H > INT32_MAX / 2) return fail(MLA_ERR_UNSUPPORTED, "too many rows");
    p.n_parts = n_parts;
    p.wire = wire ? 1 : 0;
    p.B = (int32_t)B; p.Mq = (int32_t)Mq; p.H = (int32_t)H;
    p.o_s0 = out_lat[0]->stride[0]; p.o_s1 = out_lat[0]->stride[1]; p.o_s2 = out_lat[0]->stride[2];
    p.l_s0 = out_lse[0]->stride[0]; p.l_s1 = out_lse[0]->stride[1]; p.l_s2 = out_lse[0]->stride[2];
    p.out = (float*)out->data;
    p.out_s0 = out->stride[0]; p.out_s1 = out->stride[1]; p.out_s2 = out->stride[2];
    if (merged_lse) {
      p.out_lse = (float*)merged_lse->data;
      p.ol_s0 = merged_lse->stride[0]; p.ol_s1 = merged_lse->stride[1]; p.ol_s2 = merged_lse->stride[2];
    }
    hipError_t e = mla::launch_merge(p, reinterpret_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(MLA_ERR_HIP, std::string("merge kernel launch: ") + hipGetErrorString(e));
    return MLA_OK;
  } catch (...) {
    return fail(MLA_ERR_HIP, "internal error");
  }
}

mla_status_t mla_merge_partials(const mla_tensor_t* const* out_lat,
                                const mla_tensor_t* const* out_lse, int32_t n_parts,
                                const mla_tensor_t* out, void* stream) {
  return mla_merge_partials_ex(out_lat, out_lse, n_parts, out, nullptr, stream);
}

}  // extern "C"
