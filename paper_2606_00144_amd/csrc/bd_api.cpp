// C ABI of libbd: host-side argument checks, workspace sizing and launches.
//
// Every entry point validates its arguments completely before touching the
// HIP runtime, so a rejected call launches nothing and leaves outputs alone.
// The only HIP calls made are kernel launches and hipGetLastError.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>

#include "bd.h"
#include "bd_kernels.hpp"

namespace {

thread_local char g_last_error[512] = "";

bd_status fail(bd_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return st;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Bounds on the batch shape under which every plan's arithmetic stays in range: (sequence, KV head)
// pairs and query heads per KV head.  The operations reject larger shapes as unsupported and the
// workspace-size functions answer 0 for them.
constexpr int64_t kMaxPairs = (int64_t)1 << 24;
constexpr int32_t kMaxGroup = 1 << 16;
bool shape_ok(int32_t S, int32_t Hkv, int32_t Hq) {
  return S >= 1 && Hkv >= 1 && Hq >= 1 && Hq % Hkv == 0 && (int64_t)S * Hkv <= kMaxPairs && Hq / Hkv <= kMaxGroup;
}

// Checks shared by every operation that reads the KV cache.
bd_status check_kv(const bd_kv_desc* kv, bool need_v, int32_t num_q_heads) {
  if (!kv) return fail(BD_ERR_INVALID_ARG, "kv descriptor is NULL");
  if (kv->head_dim != BD_HEAD_DIM) return fail(BD_ERR_UNSUPPORTED, "head_dim %d is not 128", kv->head_dim);
  if (!kv->k || (need_v && !kv->v)) return fail(BD_ERR_INVALID_ARG, "K or V pointer is NULL");
  if (!aligned(kv->k, 16) || (need_v && !aligned(kv->v, 16)))
    return fail(BD_ERR_INVALID_ARG, "K and V must be 16-byte aligned");
  if (!kv->seq_lens) return fail(BD_ERR_INVALID_ARG, "seq_lens is NULL");
  if (kv->num_seqs < 1 || kv->num_kv_heads < 1) return fail(BD_ERR_INVALID_ARG, "num_seqs and num_kv_heads must be >= 1");
  if (kv->max_seq_len < 0) return fail(BD_ERR_INVALID_ARG, "max_seq_len < 0");
  if (num_q_heads < 1 || num_q_heads % kv->num_kv_heads != 0)
    return fail(BD_ERR_INVALID_ARG, "num_q_heads %d is not a positive multiple of num_kv_heads %d", num_q_heads,
                kv->num_kv_heads);
  if ((int64_t)kv->num_seqs * kv->num_kv_heads > kMaxPairs || num_q_heads / kv->num_kv_heads > kMaxGroup)
    return fail(BD_ERR_UNSUPPORTED, "more than 2^24 (sequence, KV head) pairs or 2^16 query heads per KV head");
  if (kv->stride_head < 0 || kv->stride_tok < 0 || kv->stride_head % 8 || kv->stride_tok % 8)
    return fail(BD_ERR_INVALID_ARG, "stride_head and stride_tok must be non-negative multiples of 8 elements");
  if (kv->page_table) {
    if (kv->page_size < 1 || kv->max_pages_per_seq < 1 || kv->num_pages < 1)
      return fail(BD_ERR_INVALID_ARG, "paged layout needs page_size, max_pages_per_seq and num_pages >= 1");
    if ((int64_t)kv->max_seq_len > (int64_t)kv->max_pages_per_seq * kv->page_size)
      return fail(BD_ERR_INVALID_ARG, "max_seq_len exceeds max_pages_per_seq * page_size");
    if (kv->stride_page < 0 || kv->stride_page % 8)
      return fail(BD_ERR_INVALID_ARG, "stride_page must be a non-negative multiple of 8 elements");
  } else {
    if (kv->stride_seq < 0 || kv->stride_seq % 8)
      return fail(BD_ERR_INVALID_ARG, "stride_seq must be a non-negative multiple of 8 elements");
  }
  return BD_OK;
}

bd_status check_ws(void* ws, size_t have, size_t need) {
  if (need == 0) return BD_OK;
  if (!ws) return fail(BD_ERR_WORKSPACE, "workspace is NULL but %zu bytes are needed", need);
  if (!aligned(ws, 256)) return fail(BD_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (have < need) return fail(BD_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", have, need);
  return BD_OK;
}

bd_status launched(hipError_t e) {
  if (e != hipSuccess) return fail(BD_ERR_DEVICE, "launch failed: %s", hipGetErrorString(e));
  return BD_OK;
}

// ---- fixed scratch of the no-allocation entry point ---------------------------------------------
// Counter region, then split records, of bd_verify_attn_noalloc.  Each GPU the library runs on holds
// its own copy until the process ends.  In host code `scratch` only names the symbol: its device
// address comes from hipGetSymbolAddress, once per device, and only that address is passed on.
static __device__ __align__(256) uint8_t scratch[BD_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

__global__ void zero_words_kernel(uint4* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = make_uint4(0u, 0u, 0u, 0u);
}

// Device address of the current device's scratch.  The first call on a device resolves the address
// and clears the counter region with a kernel on `stream` (the calls that follow on the stream run
// after it; a completed call leaves the counters zero again).
bd_status fixed_scratch(hipStream_t stream, void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(BD_ERR_DEVICE, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(BD_ERR_UNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return fail(BD_ERR_DEVICE, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    constexpr int n = BD_WS_COUNTER_BYTES / 16;
    hipLaunchKernelGGL(zero_words_kernel, dim3(n / 256), dim3(256), 0, stream, static_cast<uint4*>(p), n);
    e = hipGetLastError();
    if (e != hipSuccess) return fail(BD_ERR_DEVICE, "clearing the scratch counters: %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return BD_OK;
}

// Largest element offset of the K/V layout plus one row; the attention kernel
// keeps row offsets as int32 in 16-byte units.
int64_t kv_extent(const bd_kv_desc* kv) {
  if (kv->page_table)
    return (int64_t)(kv->num_pages - 1) * kv->stride_page + (int64_t)(kv->num_kv_heads - 1) * kv->stride_head +
           (int64_t)(kv->page_size - 1) * kv->stride_tok + BD_HEAD_DIM;
  const int64_t L = kv->max_seq_len > 0 ? kv->max_seq_len : 1;
  return (int64_t)(kv->num_seqs - 1) * kv->stride_seq + (int64_t)(kv->num_kv_heads - 1) * kv->stride_head +
         (L - 1) * kv->stride_tok + BD_HEAD_DIM;
}

// Common launch of the attention kernel.
bd_status run_attn(const bd_kv_desc* kv, const uint16_t* q, int32_t Hq, int32_t nq, int32_t num_views,
                   const int32_t* idx, int32_t ld_idx, const int32_t* nsel, float scale, uint16_t* out_views,
                   float* lse_views, uint16_t* out_full, float* lse_full, void* ws, size_t ws_bytes,
                   hipStream_t stream, float* o32_views = nullptr, float* o32_full = nullptr,
                   bool use_fixed_scratch = false) {
  const bool train = o32_views || o32_full;
  const bd::AttnPlan pl =
      bd::plan_attn(kv->num_seqs, kv->num_kv_heads, Hq, nq, num_views, ld_idx, kv->max_seq_len, out_full != nullptr,
                    kv->page_table != nullptr, train, kv->page_table ? kv->page_size : 0);
  if (pl.block && pl.nbr > 64) return fail(BD_ERR_UNSUPPORTED, "more than 63 views with a block of more than 32 rows");
  if (pl.nblk < 0 || (!pl.block && (int64_t)pl.units_g * pl.nsplit_g + (int64_t)pl.units_f * pl.nsplit_f > INT32_MAX))
    return fail(BD_ERR_UNSUPPORTED, "problem too large for one launch");
  if (kv_extent(kv) > ((int64_t)1 << 34))
    return fail(BD_ERR_UNSUPPORTED, "K/V layout spans more than 2^34 elements");
  // counter lines: one per unit (block mode: per unit and branch), and the split kernel's group
  // counters of the two-level merge
  const int64_t lines = pl.block ? (int64_t)pl.units * pl.nbr
                                 : ((int64_t)pl.units_g + pl.units_f) * (1 + (int64_t)pl.ngrp);
  if (lines > BD_WS_COUNTER_LINES) return fail(BD_ERR_UNSUPPORTED, "more than %d work units", BD_WS_COUNTER_LINES);
  if (pl.block && (int64_t)(pl.nW + pl.nbr) * 8 * bd::attn_record_floats(2) * 4 > INT32_MAX)
    return fail(BD_ERR_UNSUPPORTED, "too many partial records per unit");
  bd_status st = BD_OK;
  if (use_fixed_scratch) {
    if (pl.ws_bytes > (size_t)BD_NOALLOC_SCRATCH_BYTES)
      return fail(BD_ERR_UNSUPPORTED, "this shape needs %zu bytes of scratch, above the fixed %d", pl.ws_bytes,
                  BD_NOALLOC_SCRATCH_BYTES);
  } else {
    st = check_ws(ws, ws_bytes, pl.ws_bytes);
    if (st != BD_OK) return st;
  }
  if (pl.nblk == 0) return BD_OK;
  if (pl.nblk >= (1 << 22)) return fail(BD_ERR_UNSUPPORTED, "more than 2^22 - 1 workgroups");
  if (use_fixed_scratch) {
    st = fixed_scratch(stream, &ws);
    if (st != BD_OK) return st;
  }
  bd::AttnParams p{};
  p.kv = bd::make_kv_view(*kv);
  p.q = q;
  p.out_g = out_views;
  p.out_f = out_full;
  p.lse_g = lse_views;
  p.lse_f = lse_full;
  p.o32_g = o32_views;
  p.o32_f = o32_full;
  p.idx = idx;
  p.nsel = nsel;
  p.ld_idx = ld_idx;
  p.S = kv->num_seqs;
  p.Hkv = kv->num_kv_heads;
  p.Hq = Hq;
  p.G = Hq / kv->num_kv_heads;
  p.nq = nq;
  p.R = pl.R;
  p.n_rb = pl.n_rb;
  p.n_rg = pl.n_rg;
  p.nsplit_g = pl.nsplit_g;
  p.kps_g = pl.kps_g;
  p.nsplit_f = pl.nsplit_f;
  p.kps_f = pl.kps_f;
  p.units_g = pl.units_g;
  p.units_all = pl.units_g + pl.units_f;
  p.ngrp = pl.ngrp;
  p.nblk_g = pl.units_g * pl.nsplit_g;
  p.page_arith = pl.page_arith ? 1 : 0;
  p.V = num_views;
  p.nbr = pl.nbr;
  p.nW = pl.nW;
  p.scale_log2 = scale * 1.4426950408889634f;
  p.max_roff = (uint32_t)((kv_extent(kv) - BD_HEAD_DIM) >> 3);
  p.counters = static_cast<uint32_t*>(ws);
  p.part = pl.record_bytes ? reinterpret_cast<float*>(static_cast<char*>(ws) + pl.counter_bytes) : nullptr;
  return launched(bd::launch_attn(p, pl, kv->page_table != nullptr, stream));
}

}  // namespace

extern "C" {

const char* bd_status_string(bd_status s) {
  switch (s) {
    case BD_OK: return "ok";
    case BD_ERR_INVALID_ARG: return "invalid argument";
    case BD_ERR_UNSUPPORTED: return "unsupported";
    case BD_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case BD_ERR_DEVICE: return "device error";
    default: return "unknown status";
  }
}

const char* bd_last_error(void) { return g_last_error; }

int32_t bd_abi_version(void) { return BD_ABI_VERSION; }

// ---------------------------------------------------------------- select
size_t bd_select_kv_workspace_bytes(int32_t num_seqs, int32_t num_kv_heads, int32_t num_q_heads, int32_t window,
                                    int32_t max_seq_len) {
  if (!shape_ok(num_seqs, num_kv_heads, num_q_heads) || window < 1 || max_seq_len < 0) return 0;
  if ((int64_t)max_seq_len - window > BD_SELECT_MAX_PREFIX || (int64_t)window * (num_q_heads / num_kv_heads) > 4096)
    return 0;
  return bd::plan_select(num_seqs, num_kv_heads, num_q_heads, window, max_seq_len, true).ws_bytes;
}

namespace {
// Common host path of both selection policies (chunk == 0: token level with pooling).
// counts_window: the budget pays for the W window positions too (B - W prefix positions), else
// for prefix positions only (B of them, B + W index slots).
bd_status run_select(const bd_kv_desc* kv, const uint16_t* q_win, int32_t num_q_heads, int32_t window, int32_t budget,
                     int32_t pool_kernel, int32_t chunk, bool counts_window, float scale, const float* lse_win,
                     int32_t* idx_out, int32_t* nsel_out, float* scores_out, void* ws, size_t ws_bytes,
                     hipStream_t stream) {
  bd_status st = check_kv(kv, false, num_q_heads);
  if (st != BD_OK) return st;
  if (window < 1 || budget < window) return fail(BD_ERR_INVALID_ARG, "need 1 <= window <= budget (window %d, budget %d)", window, budget);
  if (!counts_window && (int64_t)budget + window > INT32_MAX) return fail(BD_ERR_INVALID_ARG, "budget + window overflows");
  if (chunk < 0) return fail(BD_ERR_INVALID_ARG, "chunk must be >= 1");
  if (chunk == 0 && (pool_kernel < 1 || pool_kernel % 2 == 0))
    return fail(BD_ERR_INVALID_ARG, "pool_kernel must be odd and >= 1");
  if (chunk == 0 && pool_kernel > 255) return fail(BD_ERR_UNSUPPORTED, "pool_kernel above 255");
  if (!std::isfinite(scale) || !(scale > 0.f)) return fail(BD_ERR_INVALID_ARG, "scale must be positive and finite");
  if (!q_win || !aligned(q_win, 16)) return fail(BD_ERR_INVALID_ARG, "q_win is NULL or not 16-byte aligned");
  if (!idx_out || !nsel_out) return fail(BD_ERR_INVALID_ARG, "idx_out and nsel_out are required");
  if ((int64_t)kv->max_seq_len - window > BD_SELECT_MAX_PREFIX)
    return fail(BD_ERR_UNSUPPORTED, "max_seq_len - window exceeds %d", BD_SELECT_MAX_PREFIX);
  if ((int64_t)window * (num_q_heads / kv->num_kv_heads) > 4096)
    return fail(BD_ERR_UNSUPPORTED, "window * group above 4096 rows");
  if (kv_extent(kv) > ((int64_t)1 << 34))
    return fail(BD_ERR_UNSUPPORTED, "K layout spans more than 2^34 elements");
  const bd::SelectPlan pl = bd::plan_select(kv->num_seqs, kv->num_kv_heads, num_q_heads, window, kv->max_seq_len,
                                            kv->page_table != nullptr, kv->page_table ? kv->page_size : 0);
  st = check_ws(ws, ws_bytes, pl.ws_bytes);
  if (st != BD_OK) return st;
  bd::SelectParams p{};
  p.kv = bd::make_kv_view(*kv);
  p.q_win = q_win;
  p.lse_win = lse_win;
  p.S = kv->num_seqs;
  p.Hkv = kv->num_kv_heads;
  p.Hq = num_q_heads;
  p.G = num_q_heads / kv->num_kv_heads;
  p.W = window;
  p.budget = budget;
  p.pool_kernel = chunk > 0 ? 1 : pool_kernel;
  p.chunk = chunk;
  p.keep = counts_window ? budget - window : budget;
  p.ld = p.keep + window;
  p.R = window * p.G;
  p.n_rb = pl.n_rb;
  p.nsplit = pl.nsplit;
  p.kps = pl.kps;
  p.max_L = kv->max_seq_len;
  p.scale_log2 = scale * 1.4426950408889634f;
  p.max_roff = (uint32_t)((kv_extent(kv) - BD_HEAD_DIM) >> 3);
  char* w = static_cast<char*>(ws) + BD_WS_COUNTER_BYTES;   // the counter region stays untouched
  p.stats = reinterpret_cast<float*>(w);
  p.raw_part = reinterpret_cast<float*>(w + pl.stats_bytes);
  p.raw = scores_out;   // nullable: the total scores are exported only on request
  p.idx_out = idx_out;
  p.nsel_out = nsel_out;
  p.page_arith = pl.page_arith ? 1 : 0;
  return launched(bd::launch_select(p, kv->page_table != nullptr, stream));
}
}  // namespace

bd_status bd_select_kv(const bd_kv_desc* kv, const uint16_t* q_win, int32_t num_q_heads, int32_t window,
                       int32_t budget, int32_t pool_kernel, float scale, const float* lse_win, int32_t* idx_out,
                       int32_t* nsel_out, float* scores_out, void* ws, size_t ws_bytes, hipStream_t stream) {
  return run_select(kv, q_win, num_q_heads, window, budget, pool_kernel, 0, true, scale, lse_win, idx_out,
                    nsel_out, scores_out, ws, ws_bytes, stream);
}

bd_status bd_select_kv_chunks(const bd_kv_desc* kv, const uint16_t* q_win, int32_t num_q_heads, int32_t window,
                              int32_t budget, int32_t chunk, int32_t budget_counts_window, float scale,
                              const float* lse_win, int32_t* idx_out, int32_t* nsel_out, float* scores_out, void* ws,
                              size_t ws_bytes, hipStream_t stream) {
  if (chunk < 1) return fail(BD_ERR_INVALID_ARG, "chunk must be >= 1");
  if (budget_counts_window != 0 && budget_counts_window != 1)
    return fail(BD_ERR_INVALID_ARG, "budget_counts_window must be 0 or 1");
  return run_select(kv, q_win, num_q_heads, window, budget, 1, chunk, budget_counts_window != 0, scale, lse_win,
                    idx_out, nsel_out, scores_out, ws, ws_bytes, stream);
}

// ---------------------------------------------------------------- sparse decode
size_t bd_sparse_decode_attn_workspace_bytes(int32_t num_seqs, int32_t num_kv_heads, int32_t num_q_heads,
                                             int32_t ld_idx) {
  if (!shape_ok(num_seqs, num_kv_heads, num_q_heads) || ld_idx < 0) return 0;
  return bd::attn_ws_bytes(num_seqs, num_kv_heads, num_q_heads, 1, 1, ld_idx, 0, false);
}

bd_status bd_sparse_decode_attn(const bd_kv_desc* kv, const uint16_t* q, int32_t num_q_heads, const int32_t* idx,
                                int32_t ld_idx, const int32_t* nsel, float scale, uint16_t* out, float* lse_out,
                                void* ws, size_t ws_bytes, hipStream_t stream) {
  bd_status st = check_kv(kv, true, num_q_heads);
  if (st != BD_OK) return st;
  if (!q || !aligned(q, 16) || !out || !aligned(out, 16))
    return fail(BD_ERR_INVALID_ARG, "q and out must be non-NULL and 16-byte aligned");
  if (ld_idx < 0 || (ld_idx > 0 && (!idx || !nsel))) return fail(BD_ERR_INVALID_ARG, "idx / nsel / ld_idx invalid");
  if (!nsel) return fail(BD_ERR_INVALID_ARG, "nsel is NULL");
  if (!std::isfinite(scale) || !(scale > 0.f)) return fail(BD_ERR_INVALID_ARG, "scale must be positive and finite");
  return run_attn(kv, q, num_q_heads, 1, 1, idx, ld_idx, nsel, scale, out, lse_out, nullptr, nullptr, ws, ws_bytes,
                  stream);
}

// ---------------------------------------------------------------- multiview
size_t bd_multiview_attn_workspace_bytes(int32_t num_seqs, int32_t num_kv_heads, int32_t num_q_heads,
                                         int32_t block_len, int32_t num_views, int32_t ld_idx, int32_t max_seq_len,
                                         int32_t with_full) {
  if (!shape_ok(num_seqs, num_kv_heads, num_q_heads) || block_len < 1 || num_views < 0 || ld_idx < 0 ||
      max_seq_len < 0 || (int64_t)block_len * (num_q_heads / num_kv_heads) > (1 << 20))
    return 0;
  return bd::attn_ws_bytes(num_seqs, num_kv_heads, num_q_heads, block_len, num_views, ld_idx, max_seq_len,
                           with_full != 0, true);
}

bd_status bd_multiview_attn(const bd_kv_desc* kv, const uint16_t* q_blk, int32_t num_q_heads, int32_t block_len,
                            int32_t num_views, const int32_t* idx_views, int32_t ld_idx, const int32_t* nsel_views,
                            float scale, uint16_t* out_views, float* lse_views, float* out32_views,
                            uint16_t* out_full, float* lse_full, float* out32_full, void* ws, size_t ws_bytes,
                            hipStream_t stream) {
  bd_status st = check_kv(kv, true, num_q_heads);
  if (st != BD_OK) return st;
  if (block_len < 1 || num_views < 0 || (num_views < 1 && !out_full))
    return fail(BD_ERR_INVALID_ARG, "need block_len >= 1 and at least one view or the full branch");
  if (!q_blk || !aligned(q_blk, 16)) return fail(BD_ERR_INVALID_ARG, "q_blk is NULL or not 16-byte aligned");
  if (num_views > 0 && (!idx_views || !nsel_views || !out_views || !aligned(out_views, 16) || ld_idx < 0))
    return fail(BD_ERR_INVALID_ARG, "views need idx_views, nsel_views, ld_idx >= 0 and a 16-byte aligned out_views");
  if (out_full && !aligned(out_full, 16)) return fail(BD_ERR_INVALID_ARG, "out_full is not 16-byte aligned");
  if ((num_views > 0 && out32_views && !aligned(out32_views, 16)) || (out_full && out32_full && !aligned(out32_full, 16)))
    return fail(BD_ERR_INVALID_ARG, "out32_views and out32_full must be 16-byte aligned");
  if (!std::isfinite(scale) || !(scale > 0.f)) return fail(BD_ERR_INVALID_ARG, "scale must be positive and finite");
  if ((int64_t)block_len * (num_q_heads / kv->num_kv_heads) > (1 << 20))
    return fail(BD_ERR_UNSUPPORTED, "block_len * group too large");
  return run_attn(kv, q_blk, num_q_heads, block_len, num_views, idx_views, num_views > 0 ? ld_idx : 0, nsel_views,
                  scale, out_views, num_views > 0 ? lse_views : nullptr, out_full, out_full ? lse_full : nullptr, ws,
                  ws_bytes, stream, num_views > 0 ? out32_views : nullptr, out_full ? out32_full : nullptr);
}

// ---------------------------------------------------------------- multiview backward
size_t bd_multiview_attn_bwd_workspace_bytes(int32_t num_seqs, int32_t num_kv_heads, int32_t num_q_heads,
                                             int32_t block_len, int32_t num_views, int32_t ld_idx,
                                             int32_t max_seq_len, int32_t with_full) {
  if (!shape_ok(num_seqs, num_kv_heads, num_q_heads) || block_len < 1 || block_len > bd::kMaxBwdBlock ||
      num_views < 0 || num_views > 64 - (with_full != 0 ? 1 : 0) || ld_idx < 0 || max_seq_len < 0 ||
      (int64_t)block_len * (num_q_heads / num_kv_heads) > (1 << 20))
    return 0;
  const int32_t ld = num_views > 0 ? ld_idx : 0;
  return bd::plan_attn_bwd(num_seqs, num_kv_heads, num_q_heads, block_len, num_views, ld, max_seq_len,
                           with_full != 0, true).ws_bytes;
}

bd_status bd_multiview_attn_bwd(const bd_kv_desc* kv, const uint16_t* q_blk, int32_t num_q_heads, int32_t block_len,
                                int32_t num_views, const int32_t* idx_views, int32_t ld_idx,
                                const int32_t* nsel_views, float scale, const float* out32_views,
                                const float* lse_views, const uint16_t* dout_views, const float* out32_full,
                                const float* lse_full, const uint16_t* dout_full, float* dq, float* dk_blk,
                                float* dv_blk, void* ws, size_t ws_bytes, hipStream_t stream) {
  bd_status st = check_kv(kv, true, num_q_heads);
  if (st != BD_OK) return st;
  const bool full = dout_full != nullptr;
  if (block_len < 1 || num_views < 0 || (num_views < 1 && !full))
    return fail(BD_ERR_INVALID_ARG, "need block_len >= 1 and at least one view or the full branch");
  if (block_len > bd::kMaxBwdBlock) return fail(BD_ERR_UNSUPPORTED, "block_len above %d", bd::kMaxBwdBlock);
  if ((int64_t)block_len * (num_q_heads / kv->num_kv_heads) > (1 << 20))
    return fail(BD_ERR_UNSUPPORTED, "block_len * group too large");
  if (!q_blk || !aligned(q_blk, 16)) return fail(BD_ERR_INVALID_ARG, "q_blk is NULL or not 16-byte aligned");
  if (num_views > 0 && (!idx_views || !nsel_views || ld_idx < 0 || !out32_views || !aligned(out32_views, 16) ||
                        !lse_views || !dout_views || !aligned(dout_views, 16)))
    return fail(BD_ERR_INVALID_ARG,
                "views need idx_views, nsel_views, ld_idx >= 0, lse_views and 16-byte aligned out32_views, dout_views");
  if ((out32_full != nullptr) != full || (lse_full != nullptr) != full)
    return fail(BD_ERR_INVALID_ARG, "out32_full, lse_full and dout_full must be all NULL or all given");
  if (full && (!aligned(out32_full, 16) || !aligned(dout_full, 16)))
    return fail(BD_ERR_INVALID_ARG, "out32_full and dout_full must be 16-byte aligned");
  if (!dq || !aligned(dq, 16)) return fail(BD_ERR_INVALID_ARG, "dq is NULL or not 16-byte aligned");
  if ((dk_blk != nullptr) != (dv_blk != nullptr) || (dk_blk && (!aligned(dk_blk, 16) || !aligned(dv_blk, 16))))
    return fail(BD_ERR_INVALID_ARG, "dk_blk and dv_blk must be both NULL or both given, 16-byte aligned");
  if (!std::isfinite(scale) || !(scale > 0.f)) return fail(BD_ERR_INVALID_ARG, "scale must be positive and finite");
  if (kv_extent(kv) > ((int64_t)1 << 34))
    return fail(BD_ERR_UNSUPPORTED, "K/V layout spans more than 2^34 elements");
  const int32_t ld = num_views > 0 ? ld_idx : 0;
  const bool paged = kv->page_table != nullptr;
  const bd::AttnBwdPlan pl = bd::plan_attn_bwd(kv->num_seqs, kv->num_kv_heads, num_q_heads, block_len, num_views, ld,
                                               kv->max_seq_len, full, dk_blk != nullptr);
  if ((int64_t)pl.units + (int64_t)kv->num_seqs * kv->num_kv_heads > BD_WS_COUNTER_LINES)
    return fail(BD_ERR_UNSUPPORTED, "more than %d work units", BD_WS_COUNTER_LINES);
  if (pl.nbr > 64) return fail(BD_ERR_UNSUPPORTED, "more than 64 branches (views and the full cache)");
  if ((int64_t)pl.units * pl.nW > INT32_MAX / 2 || (int64_t)pl.nW * 2 * 16 * BD_HEAD_DIM * 4 > INT32_MAX ||
      (int64_t)pl.nbr * block_len * 2 * BD_HEAD_DIM * 4 > INT32_MAX ||
      (int64_t)kv->num_seqs * kv->num_kv_heads * pl.nbr > INT32_MAX / 2)
    return fail(BD_ERR_UNSUPPORTED, "problem too large for one launch");
  st = check_ws(ws, ws_bytes, pl.ws_bytes);
  if (st != BD_OK) return st;
  bd::AttnBwdParams p{};
  p.kv = bd::make_kv_view(*kv);
  p.q = q_blk;
  p.o32_g = out32_views;
  p.lse_g = lse_views;
  p.dout_g = dout_views;
  p.o32_f = out32_full;
  p.lse_f = lse_full;
  p.dout_f = dout_full;
  p.idx = idx_views;
  p.nsel = nsel_views;
  p.ld_idx = ld;
  p.S = kv->num_seqs;
  p.Hkv = kv->num_kv_heads;
  p.Hq = num_q_heads;
  p.G = num_q_heads / kv->num_kv_heads;
  p.C = block_len;
  p.V = num_views;
  p.inv_G = 1.f / (float)p.G;
  p.R = pl.R;
  p.n_rb = pl.n_rb;
  p.n_rg = pl.n_rg;
  p.nW = pl.nW;
  p.units = pl.units;
  p.nbr = pl.nbr;
  p.nkt = pl.nkt;
  p.scale = scale;
  p.scale_log2 = scale * 1.4426950408889634f;
  p.max_roff = (uint32_t)((kv_extent(kv) - BD_HEAD_DIM) >> 3);
  p.dq = dq;
  p.dk = dk_blk;
  p.dv = dv_blk;
  char* w = static_cast<char*>(ws);
  p.counters = reinterpret_cast<uint32_t*>(w);
  p.part_q = pl.q_record_bytes ? reinterpret_cast<float*>(w + pl.counter_bytes) : nullptr;
  p.part_kv = pl.kv_record_bytes ? reinterpret_cast<float*>(w + pl.counter_bytes + pl.q_record_bytes) : nullptr;
  p.rstats = pl.d_bytes ? reinterpret_cast<float*>(w + pl.counter_bytes + pl.q_record_bytes + pl.kv_record_bytes)
                        : nullptr;
  p.R_pad = pl.R_pad;
  return launched(bd::launch_attn_bwd(p, pl, paged, stream));
}

// ---------------------------------------------------------------- verify
size_t bd_verify_attn_workspace_bytes(int32_t num_seqs, int32_t num_kv_heads, int32_t num_q_heads, int32_t gamma,
                                      int32_t max_seq_len) {
  if (!shape_ok(num_seqs, num_kv_heads, num_q_heads) || gamma < 0 || gamma > 4095 || max_seq_len < 0) return 0;
  return bd::attn_ws_bytes(num_seqs, num_kv_heads, num_q_heads, gamma + 1, 0, 0, max_seq_len, true);
}

namespace {
bd_status check_verify(const bd_kv_desc* kv, const uint16_t* q, int32_t num_q_heads, int32_t gamma, float scale,
                       const uint16_t* out) {
  bd_status st = check_kv(kv, true, num_q_heads);
  if (st != BD_OK) return st;
  if (gamma < 0 || gamma > 4095) return fail(BD_ERR_INVALID_ARG, "gamma %d outside [0, 4095]", gamma);
  if (!q || !aligned(q, 16) || !out || !aligned(out, 16))
    return fail(BD_ERR_INVALID_ARG, "q and out must be non-NULL and 16-byte aligned");
  if (!std::isfinite(scale) || !(scale > 0.f)) return fail(BD_ERR_INVALID_ARG, "scale must be positive and finite");
  return BD_OK;
}
}  // namespace

bd_status bd_verify_attn(const bd_kv_desc* kv, const uint16_t* q, int32_t num_q_heads, int32_t gamma, float scale,
                         uint16_t* out, float* lse_out, void* ws, size_t ws_bytes, hipStream_t stream) {
  const bd_status st = check_verify(kv, q, num_q_heads, gamma, scale, out);
  if (st != BD_OK) return st;
  return run_attn(kv, q, num_q_heads, gamma + 1, 0, nullptr, 0, nullptr, scale, nullptr, nullptr, out, lse_out, ws,
                  ws_bytes, stream);
}

bd_status bd_verify_attn_noalloc(const bd_kv_desc* kv, const uint16_t* q, int32_t num_q_heads, int32_t gamma,
                                 float scale, uint16_t* out, float* lse_out, hipStream_t stream) {
  const bd_status st = check_verify(kv, q, num_q_heads, gamma, scale, out);
  if (st != BD_OK) return st;
  return run_attn(kv, q, num_q_heads, gamma + 1, 0, nullptr, 0, nullptr, scale, nullptr, nullptr, out, lse_out,
                  nullptr, 0, stream, nullptr, nullptr, true);
}

// ---------------------------------------------------------------- accept
size_t bd_accept_len_workspace_bytes(int32_t num_seqs, int32_t gamma, int32_t vocab) {
  if (num_seqs < 1 || gamma < 0 || gamma > 63 || vocab < 1) return 0;
  return bd::plan_accept(num_seqs, gamma, vocab).ws_bytes;
}

bd_status bd_accept_len(const float* logits, int64_t row_stride, const int32_t* draft, int32_t num_seqs, int32_t gamma,
                        int32_t vocab, int32_t* accept_out, int32_t* bonus_out, int32_t* argmax_out, void* ws,
                        size_t ws_bytes, hipStream_t stream) {
  if (!logits || !accept_out) return fail(BD_ERR_INVALID_ARG, "logits and accept_out are required");
  if (num_seqs < 1 || vocab < 1 || gamma < 0) return fail(BD_ERR_INVALID_ARG, "need num_seqs >= 1, vocab >= 1, gamma >= 0");
  if (gamma > 63) return fail(BD_ERR_UNSUPPORTED, "gamma above 63");
  if (gamma > 0 && !draft) return fail(BD_ERR_INVALID_ARG, "draft is NULL");
  if (row_stride < vocab) return fail(BD_ERR_INVALID_ARG, "row_stride %lld < vocab %d", (long long)row_stride, vocab);
  if ((int64_t)num_seqs * (gamma + 1) * 1024 > INT32_MAX) return fail(BD_ERR_UNSUPPORTED, "too many rows");
  if ((int64_t)num_seqs * (2 * gamma + 3) > BD_WS_COUNTER_LINES)
    return fail(BD_ERR_UNSUPPORTED, "more than %d sequence and row counter lines", BD_WS_COUNTER_LINES);
  const bd::AcceptPlan pl = bd::plan_accept(num_seqs, gamma, vocab);
  if ((int64_t)num_seqs * (gamma + 1) * pl.nsplit >= (1 << 22))
    return fail(BD_ERR_UNSUPPORTED, "more than 2^22 - 1 workgroups");
  bd_status st = check_ws(ws, ws_bytes, pl.ws_bytes);
  if (st != BD_OK) return st;
  bd::AcceptParams p{};
  p.logits = logits;
  p.row_stride = row_stride;
  p.draft = draft;
  p.S = num_seqs;
  p.gamma = gamma;
  p.vocab = vocab;
  p.nsplit = pl.nsplit;
  p.chunk = pl.chunk;
  p.vec4 = aligned(logits, 16) && (row_stride % 4 == 0);
  p.accept_out = accept_out;
  p.bonus_out = bonus_out;
  p.argmax_out = argmax_out;
  p.counters = static_cast<uint32_t*>(ws);
  return launched(bd::launch_accept(p, stream));
}

// ---------------------------------------------------------------- per-round cache updates
bd_status bd_cache_append(const bd_kv_desc* kv, const uint16_t* k_new, const uint16_t* v_new, int32_t n,
                          int32_t* idx, int32_t ld_idx, int32_t* nsel, hipStream_t stream) {
  bd_status st = check_kv(kv, true, kv ? kv->num_kv_heads : 0);
  if (st != BD_OK) return st;
  if (n < 0) return fail(BD_ERR_INVALID_ARG, "n < 0");
  if (n == 0) return BD_OK;
  if (!k_new || !v_new || !aligned(k_new, 16) || !aligned(v_new, 16))
    return fail(BD_ERR_INVALID_ARG, "k_new and v_new must be 16-byte aligned device pointers");
  if ((idx == nullptr) != (nsel == nullptr)) return fail(BD_ERR_INVALID_ARG, "idx and nsel go together");
  if (idx && ld_idx < 0) return fail(BD_ERR_INVALID_ARG, "ld_idx < 0");
  if ((int64_t)kv->num_seqs * n > INT32_MAX) return fail(BD_ERR_UNSUPPORTED, "num_seqs * n too large");
  bd::AppendParams p{};
  p.kv = bd::make_kv_view(*kv);
  p.k_new = k_new;
  p.v_new = v_new;
  p.n = n;
  p.idx = idx;
  p.nsel = nsel;
  p.ld_idx = idx ? ld_idx : 0;
  return launched(bd::launch_append(p, stream));
}

bd_status bd_cache_rollback(int32_t* seq_lens, int32_t* nsel, const int32_t* accept, int32_t num_seqs, int32_t spec,
                            const int32_t* base_lens, const int32_t* base_nsel, hipStream_t stream) {
  if (!seq_lens || !accept) return fail(BD_ERR_INVALID_ARG, "seq_lens and accept are required");
  if (num_seqs < 1 || spec < 0) return fail(BD_ERR_INVALID_ARG, "need num_seqs >= 1 and spec >= 0");
  if (base_nsel && !nsel) return fail(BD_ERR_INVALID_ARG, "base_nsel without nsel");
  bd::RollbackParams p{seq_lens, nsel, accept, base_lens, base_nsel, num_seqs, spec};
  return launched(bd::launch_rollback(p, stream));
}

// ---------------------------------------------------------------- top-1 CE, budget sampling
size_t bd_top1_ce_workspace_bytes(int32_t rows, int32_t vocab) {
  if (rows < 1 || vocab < 1) return 0;
  return bd::plan_ce(rows, vocab).ws_bytes;
}

bd_status bd_top1_ce(const float* student, int64_t student_stride, const float* teacher, int64_t teacher_stride,
                     const int32_t* targets, int32_t rows, int32_t vocab, float* loss_out, int32_t* target_out,
                     float* lse_out, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!student || !loss_out) return fail(BD_ERR_INVALID_ARG, "student and loss_out are required");
  if ((teacher == nullptr) == (targets == nullptr)) return fail(BD_ERR_INVALID_ARG, "give exactly one of teacher and targets");
  if (rows < 1 || vocab < 1) return fail(BD_ERR_INVALID_ARG, "need rows >= 1 and vocab >= 1");
  if (student_stride < vocab || (teacher && teacher_stride < vocab))
    return fail(BD_ERR_INVALID_ARG, "row strides must be >= vocab");
  if (rows > BD_WS_COUNTER_LINES) return fail(BD_ERR_UNSUPPORTED, "more than %d rows", BD_WS_COUNTER_LINES);
  const bd::CePlan pl = bd::plan_ce(rows, vocab);
  if ((int64_t)rows * pl.nsplit > INT32_MAX) return fail(BD_ERR_UNSUPPORTED, "too many rows");
  bd_status st = check_ws(ws, ws_bytes, pl.ws_bytes);
  if (st != BD_OK) return st;
  bd::CeParams p{};
  p.student = student;
  p.s_stride = student_stride;
  p.teacher = teacher;
  p.t_stride = teacher ? teacher_stride : 0;
  p.targets = targets;
  p.rows = rows;
  p.vocab = vocab;
  p.nsplit = pl.nsplit;
  p.chunk = pl.chunk;
  p.vec4 = aligned(student, 16) && student_stride % 4 == 0 && (!teacher || (aligned(teacher, 16) && teacher_stride % 4 == 0));
  p.loss_out = loss_out;
  p.target_out = target_out;
  p.lse_out = lse_out;
  p.counters = static_cast<uint32_t*>(ws);
  p.part = reinterpret_cast<float*>(static_cast<char*>(ws) + BD_WS_COUNTER_BYTES);
  return launched(bd::launch_ce(p, stream));
}

bd_status bd_sample_budgets(const float* u, int32_t count, const int32_t* budgets, const float* weights, int32_t n,
                            int32_t* out, hipStream_t stream) {
  if (!u || !out || !budgets || !weights) return fail(BD_ERR_INVALID_ARG, "u, budgets, weights and out are required");
  if (count < 0 || n < 1 || n > bd::kMaxBudgets) return fail(BD_ERR_INVALID_ARG, "need count >= 0 and 1 <= n <= %d", bd::kMaxBudgets);
  bd::SampleTable t{};
  t.n = n;
  float acc = 0.f;
  for (int i = 0; i < n; ++i) {
    if (!std::isfinite(weights[i]) || !(weights[i] > 0.f)) return fail(BD_ERR_INVALID_ARG, "weights must be positive and finite");
    acc += weights[i];
    t.thr[i] = acc;
    t.budgets[i] = budgets[i];
  }
  for (int i = 0; i < n; ++i) t.thr[i] = t.thr[i] / acc;
  if (count == 0) return BD_OK;
  return launched(bd::launch_sample(u, count, t, out, stream));
}

}  // extern "C"
