// Kernel parameter blocks and launchers of libbd (shared by the host API and the kernels).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "bd_common.hpp"

namespace bd {

// Largest number of keys one attention workgroup takes through its slot table (gathered
// entries, or cache rows of a paged cache).
constexpr int kMaxSplitKeys = 2048;

// ---- attention (decode / verify / multiview) -------------------------------
struct AttnParams {
  KvView kv;
  const uint16_t* q;        // [S][nq][Hq][D]
  uint16_t* out_g;          // gathered views: [V][S][nq][Hq][D]
  uint16_t* out_f;          // full branch: [S][nq][Hq][D]
  float* lse_g;             // nullable [V][S][nq][Hq]
  float* lse_f;             // nullable [S][nq][Hq]
  float* o32_g;             // nullable fp32 outputs of the views (block mode only; selects the two-term weights)
  float* o32_f;             // nullable fp32 output of the full branch (block mode only)
  const int32_t* idx;       // [V][S][Hkv][ld_idx]
  const int32_t* nsel;      // [V][S]
  int32_t ld_idx;
  int32_t S, Hkv, Hq, G;
  int32_t nq;               // query rows per head (1, gamma+1 or C)
  int32_t R;                // rows per (s, g): nq * G
  int32_t n_rb;             // row blocks of 16*NT rows
  int32_t n_rg;             // block mode: row groups of 8 row blocks (otherwise n_rb)
  int32_t nsplit_g, kps_g;  // gathered units: splits and entries per split
  int32_t nsplit_f, kps_f;  // full units: splits and keys per split
  int32_t units_g;          // gathered units (their blocks come first)
  int32_t units_all;        // gathered and full units: counter lines 0 .. units_all-1
  int32_t ngrp;             // two-level merge: group counter lines per unit (0 when no unit needs them)
  int32_t nblk_g;           // blocks of gathered units
  int32_t V, nbr;           // block mode: views, and branches (views + full)
  int32_t nW;               // block mode: workgroups per (s, g, row group), equal shares of its key stream
  int32_t nblk;             // workgroups of the launch (set by launch_attn)
  float scale_log2;         // softmax scale * log2(e)
  uint32_t max_roff;        // largest valid row offset of the K/V layout, 16-byte units
  float* part;              // partial records
  uint32_t* counters;       // one per unit
  int32_t page_arith;       // 1: the full branch of the paged cache reads its rows through a table of page offsets
};

struct AttnPlan {
  int nt, n_rb, R;
  bool block;               // block mode: 8 waves, one 32-row block each, sharing every K/V tile
  int n_rg;
  int nsplit_g, kps_g, nsplit_f, kps_f;
  int units_g, units_f, nblk;
  int ngrp;                 // group counters per unit of the two-level split merge (0: none)
  bool page_arith;          // paged full branch through the table of page offsets (pages of 16k rows)
  int units, nbr, nW;       // block mode: (s, g, row group) units, branches, workgroups per unit
  size_t counter_bytes, record_bytes, ws_bytes;
};

// `paged`: the cache is paged.  Its full branch goes through a table that bounds the splits: one
// entry per key, or with `page_size` a multiple of 16 (pages hold whole 16-key sub-tiles) one entry
// per page, which bounds them far less.  `train`: fp32 outputs are requested (block mode with
// two-term weights).  Workspace queries that do not know the layout take the largest of the plans
// (attn_ws_bytes: the per-key table's plan, which never needs less scratch than the per-page one).
AttnPlan plan_attn(int S, int Hkv, int Hq, int nq, int num_views, int ld_idx, int max_L, bool with_full, bool paged,
                   bool train = false, int page_size = 0);
hipError_t launch_attn(const AttnParams& p, const AttnPlan& pl, bool paged, hipStream_t stream);
size_t attn_record_floats(int nt);
// Workspace bytes that serve either layout (paged or contiguous) of the given shape, and with
// train_capable also the training outputs.
size_t attn_ws_bytes(int S, int Hkv, int Hq, int nq, int num_views, int ld_idx, int max_L, bool with_full,
                     bool train_capable = false);

// ---- multiview attention backward -------------------------------------------
// Branch b of a (sequence, KV head) pair is view b (b < V) or the full cache (b == V).
constexpr int kMaxBwdBlock = 1024;   // largest block C the backward accepts (key counts live in LDS)

struct AttnBwdParams {
  KvView kv;
  const uint16_t* q;         // [S][C][Hq][D]
  const float* o32_g;        // views: fp32 forward outputs [V][S][C][Hq][D]
  const float* lse_g;        // views: log-sum-exp [V][S][C][Hq]
  const uint16_t* dout_g;    // views: upstream gradients [V][S][C][Hq][D]
  const float* o32_f;        // full branch (NULL: none)
  const float* lse_f;
  const uint16_t* dout_f;
  const int32_t* idx;        // [V][S][Hkv][ld_idx]
  const int32_t* nsel;       // [V][S]
  int32_t ld_idx;
  int32_t S, Hkv, Hq, G, C, V;
  int32_t R;                 // rows per (s, g): C * G
  int32_t n_rb, n_rg;        // 32-row blocks, groups of 8 of them
  int32_t nW;                // dQ workgroups per unit, each a share of the unit's key stream
  int32_t units;             // S * Hkv * n_rg (dQ units; their counters come first)
  int32_t nbr;               // branches: V + (full ? 1 : 0)
  int32_t nkt;               // 16-key tiles of the block
  float scale, scale_log2;
  float inv_G;               // 1 / G
  uint32_t max_roff;         // largest valid row offset of the K/V layout, 16-byte units
  float* dq;                 // [S][C][Hq][D]
  float* dk;                 // nullable [S][C][Hkv][D] (with dv)
  float* dv;
  float* part_q;             // dQ partial records: [unit][wave][nW] of 32 x 128
  float* part_kv;            // dK/dV partial records: [(s, g)][branch] of C x (dK | dV) x 128
  float* rstats;             // with dK/dV: per branch row (lse in log2 units, D = <dO, O>),
                             // [nbr][S * Hkv][R_pad][2], published by the dQ kernel
  int32_t R_pad;             // rows rounded up to 32
  uint32_t* counters;
};

struct AttnBwdPlan {
  int n_rb, n_rg, R, R_pad, units, nbr, nkt, nW, nblk_q, nblk_kv;
  size_t counter_bytes, q_record_bytes, kv_record_bytes, d_bytes, ws_bytes;
};

AttnBwdPlan plan_attn_bwd(int S, int Hkv, int Hq, int C, int num_views, int ld_idx, int max_L, bool with_full,
                          bool with_dkv);
hipError_t launch_attn_bwd(const AttnBwdParams& p, const AttnBwdPlan& pl, bool paged, hipStream_t stream);

// ---- greedy acceptance -----------------------------------------------------
struct AcceptParams {
  const float* logits;
  int64_t row_stride;
  const int32_t* draft;
  int32_t S, gamma, vocab;
  int32_t nsplit, chunk;    // vocab chunks per row and floats per chunk
  int32_t vec4;             // rows 16-byte aligned: vector loads
  int32_t nblk;             // workgroups of the launch (set by launch_accept)
  int32_t* accept_out;
  int32_t* bonus_out;
  int32_t* argmax_out;
  // counter region lines: [S] sequence counters, [S][gamma+1] row counters, then [S][gamma+1]
  // row maxima (packed keys, max-combined by the row's chunks)
  uint32_t* counters;
};

struct AcceptPlan {
  int nsplit, chunk;
  size_t counter_bytes, ws_bytes;
};

AcceptPlan plan_accept(int S, int gamma, int vocab);
hipError_t launch_accept(const AcceptParams& p, hipStream_t stream);

// ---- budgeted selection ----------------------------------------------------
struct SelectParams {
  KvView kv;
  const uint16_t* q_win;    // [S][W][Hq][D]
  const float* lse_win;     // nullable [S][W][Hq]
  int32_t S, Hkv, Hq, G, W;
  int32_t budget, pool_kernel;
  int32_t chunk;            // 0: token-level selection with pooling; > 0: TopKChunks with this chunk size
  int32_t keep;             // prefix positions the budget pays for: budget - W, or budget (B excludes the window)
  int32_t ld;               // index slots per (s, g): keep + W
  int32_t R;                // rows per (s, g): W * G
  int32_t n_rb;             // row blocks of 16*NT rows
  int32_t nsplit, kps;      // key splits of the scoring passes
  int32_t max_L;
  float scale_log2;
  uint32_t max_roff;        // largest valid row offset of the K layout, 16-byte units
  float* stats;             // [S][Hkv][n_rb][nsplit][128][2] per-split row max / sum
  float* raw_part;          // [S][Hkv][n_rb][max_L] per-row-block column sums
  float* raw;               // nullable [S][Hkv][max_L] total raw scores (the caller's scores_out)
  int32_t* idx_out;         // [S][Hkv][ld]
  int32_t* nsel_out;        // [S]
  int32_t page_arith;       // 1: paged rows through a table of page offsets (pages of 16k rows)
};

struct SelectPlan {
  int n_rb, nsplit, kps;
  bool page_arith;          // paged splits through the table of page offsets
  size_t stats_bytes, raw_part_bytes, ws_bytes;
};

// `paged`: the cache is paged; its splits then go through a table of bounded size, with one entry per
// key, or with `page_size` a multiple of 16 (pages hold whole 16-key sub-tiles) one per page.
// Workspace queries that do not know the layout use paged = true with the per-key table, which has
// at least as many splits.
SelectPlan plan_select(int S, int Hkv, int Hq, int W, int max_L, bool paged, int page_size = 0);
hipError_t launch_select(const SelectParams& p, bool paged, hipStream_t stream);

// ---- per-round cache updates -------------------------------------------------
struct AppendParams {
  KvView kv;                // the cache written (k, v rows; seq_lens advanced in place)
  const uint16_t* k_new;    // [S][n][Hkv][D]
  const uint16_t* v_new;
  int32_t n;
  int32_t* idx;             // nullable [S][Hkv][ld_idx] sparse list, entries appended
  int32_t* nsel;            // [S] when idx is given
  int32_t ld_idx;
};

hipError_t launch_append(const AppendParams& p, hipStream_t stream);
struct RollbackParams {
  int32_t* seq_lens;        // [S], updated in place
  int32_t* nsel;            // nullable [S], updated in place
  const int32_t* accept;    // [S]
  const int32_t* base_lens; // nullable [S]: lengths before the speculative appends
  const int32_t* base_nsel; // nullable [S]: list counts before them
  int32_t S, spec;
};
hipError_t launch_rollback(const RollbackParams& p, hipStream_t stream);

// ---- top-1 cross-entropy and budget sampling ---------------------------------
struct CeParams {
  const float* student;     // [rows] rows of vocab fp32 at s_stride
  int64_t s_stride;
  const float* teacher;     // nullable [rows] rows at t_stride: targets = first argmax
  int64_t t_stride;
  const int32_t* targets;   // [rows] when teacher is NULL
  int32_t rows, vocab;
  int32_t nsplit, chunk;
  int32_t vec4;             // both row sets 16-byte aligned: vector loads
  float* loss_out;
  int32_t* target_out;      // nullable
  float* lse_out;           // nullable
  float* part;              // [rows][nsplit] 16-byte chunk records
  uint32_t* counters;       // counter region: one line per row
};

struct CePlan {
  int nsplit, chunk;
  size_t record_bytes, ws_bytes;
};

CePlan plan_ce(int rows, int vocab);
hipError_t launch_ce(const CeParams& p, hipStream_t stream);

constexpr int kMaxBudgets = 16;
struct SampleTable {
  int32_t n;
  int32_t budgets[kMaxBudgets];
  float thr[kMaxBudgets];   // fp32 cumulative thresholds, the last one 1
};
hipError_t launch_sample(const float* u, int32_t count, const SampleTable& t, int32_t* out, hipStream_t stream);

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

}  // namespace bd
