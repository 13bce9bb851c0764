// Tile-streaming pieces shared by the attention kernels (forward and backward).
#pragma once

#include "bd_common.hpp"

namespace bd {

template <bool B>
struct BoolTag { static constexpr bool value = B; };

// One 16-byte direct-to-LDS load (global_load_lds_dwordx4): lane l's bytes land at the
// wave's LDS base + 16*l.
__device__ inline void dma16(const uint16_t* g, uint8_t* l) {
  __builtin_amdgcn_global_load_lds((const void*)g, (__attribute__((address_space(3))) void*)l, 16, 0, 0);
}
// The same with the non-temporal policy (nt), for data read once per call.
constexpr int kPolicyNt = 2;
__device__ inline void dma16_nt(const uint16_t* g, uint8_t* l) {
  __builtin_amdgcn_global_load_lds((const void*)g, (__attribute__((address_space(3))) void*)l, 16, 0, kPolicyNt);
}

// Transposed operand for d-tile dt from 8 rows of 16 bytes per lane (row slot i = register i,
// bytes 16*(lane%16) of the row): slot i of the result holds row i's element 8*(lane%16) + dt.
// An 8x8 bf16 block transposed in registers with byte permutes.
__device__ inline bf16x8 vt_operand(const u32x4 (&v)[8], int dt) {
  const int w = dt >> 1;
  const uint32_t sel = (dt & 1) ? 0x07060302u : 0x05040100u;
  u32x4 r;
  r[0] = __builtin_amdgcn_perm(v[1][w], v[0][w], sel);
  r[1] = __builtin_amdgcn_perm(v[3][w], v[2][w], sel);
  r[2] = __builtin_amdgcn_perm(v[5][w], v[4][w], sel);
  r[3] = __builtin_amdgcn_perm(v[7][w], v[6][w], sel);
  return as_bf16x8(r);
}

// Slot table of one split for the block-mode kernels: row offset (16-byte units) and position of
// every key slot in [0, nslots), entries e_begin .. e_end-1 of the key list (gathered idx entries,
// or cache rows when idx_row is NULL) followed by padding slots (position -1, offset 0).  Keys
// outside [0, L) and rows whose page is outside the pool become padding too.  All idx and
// page-table loads are issued before any result is used.
template <bool PAGED, int kThreadsT, int kCap>
__device__ inline void fill_slot_table(const KvView& kv, int s, int g, int L, const int32_t* idx_row, int e_begin,
                                       int e_end, int nslots, int32_t* roff, int32_t* tpos, int tid) {
  constexpr int kPer = (kCap + kThreadsT - 1) / kThreadsT;
  int tv[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int e = e_begin + tid + k * kThreadsT;
    int t = -1;
    if (e < e_end) t = idx_row ? idx_row[e] : e;
    tv[k] = (t >= 0 && t < L) ? t : -1;
  }
  int pg[kPer];
  if constexpr (PAGED) {
#pragma unroll
    for (int k = 0; k < kPer; ++k)
      pg[k] = tv[k] >= 0 ? kv.page_table[(int64_t)s * kv.max_pages_per_seq + tv[k] / kv.page_size] : 0;
  }
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int i = tid + k * kThreadsT;
    if (i < nslots && i < kCap) {
      int t = tv[k];
      int64_t o;
      if constexpr (PAGED) {
        o = (unsigned)pg[k] < (unsigned)kv.num_pages
                ? (int64_t)pg[k] * kv.stride_page + (int64_t)g * kv.stride_head +
                      (int64_t)(t % kv.page_size) * kv.stride_tok
                : -1;
      } else {
        o = (int64_t)s * kv.stride_seq + (int64_t)g * kv.stride_head + (int64_t)t * kv.stride_tok;
      }
      if (t < 0 || o < 0) { t = -1; o = 0; }
      roff[i] = (int)(o >> 3);
      tpos[i] = t;
    }
  }
}

// How a (sequence, KV head, row group) unit's key stream (the views' entry lists, then the full
// branch's cache rows) is cut among its nW workgroups: equal shares of weighted work, a gathered
// view entry weighing WG and a cache row of the full branch WF (gathered tiles cost more per tile).
// Views come first, so stream position x (vt = the views' total) weighs WG*x up to vt and WF per
// row after.  A share weighs at least WG*32, so every workgroup below the stream's end gets entries
// and the workgroups that meet a branch are consecutive.  All kernels over a unit's stream cut it
// with the same weights.
// ROUND: the share's weight is rounded up to a multiple of ROUND (with WG = WF = 1 and ROUND = 32,
// equal shares that start on whole tiles of the stream).
template <int WG, int WF, int ROUND = 1>
struct StreamCut {
  int vt, total, chunk;   // chunk: weight per workgroup
  __device__ StreamCut(int vt_, int total_, int nW) : vt(vt_), total(total_) {
    const int tw = WG * vt + WF * (total - vt);
    int c = (tw + nW - 1) / nW;
    c = (c + ROUND - 1) / ROUND * ROUND;
    chunk = c > WG * 32 ? c : WG * 32;
  }
  __device__ int weight(int x) const { return x <= vt ? WG * x : WG * vt + WF * (x - vt); }
  // workgroup whose share holds stream position x
  __device__ int wg_of(int x) const { return weight(x) / chunk; }
  // first stream position of workgroup w's share (clamped to the stream's end)
  __device__ int start_of(int w) const {
    const int t = w * chunk;
    const int x = t <= WG * vt ? (t + WG - 1) / WG : vt + (t - WG * vt + WF - 1) / WF;
    return x < total ? x : total;
  }
};
// Most entries a share can hold: chunk / WF + 1 with chunk = ceil(weighted total / nW); the
// smallest nW keeping that within `cap` for a stream of at most stream_max entries.
template <int WG, int WF>
inline int64_t stream_cut_min_workgroups(int64_t stream_max, int cap) {
  const int64_t per = (int64_t)WF * (cap - 32);
  return (WG * stream_max + per - 1) / per;
}

}  // namespace bd
