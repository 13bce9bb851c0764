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

// A tile of 32 key rows kept row-major for the transposing reads: load q (0..7) of lane l brings
// row 4*q + l/16, its 16-byte chunk (l%16) ^ (l/16), to byte rm_block_off(q) + 256*(l/16) +
// 16*(l%16), so chunk c of row r sits at position c ^ (r % 4) and a 16-lane group's reads cover
// 32 distinct banks.  The LDS serves a transposing read 32 lanes (64 banks of 4 bytes) at a time,
// and lanes 0-15 and 16-31 read rows of consecutive blocks (1 KiB, rows 4q .. 4q+3).  At a 1 KiB
// pitch both lane groups meet on the same 32 banks: an in-bounds probe measured every read 2-way
// conflicted.  So odd blocks start 8 bytes past a 16-byte boundary (the other 32 banks), and every
// pair of blocks takes 16 bytes more so that the shifted block does not run into the next: block q
// at 1024*q + 8*(q%2) + 16*(q/2).  The probe then read every element where the layout below says
// and measured no conflict (40% less time).  Rows 16..31 (blocks 4..7) lie 4128 bytes past rows 0..15.
constexpr int kRmTileBytes = 8256;
constexpr int kRmHighRows = 4128;
__device__ inline uint32_t rm_block_off(int q) {
  return 1024u * (uint32_t)q + 8u * (uint32_t)(q & 1) + 16u * (uint32_t)(q >> 1);
}
__device__ inline int rm_row(int q, int lane) { return 4 * q + (lane >> 4); }
__device__ inline int rm_chunk(int lane) { return (lane & 15) ^ (lane >> 4); }
// This lane's read_vt_tr addresses relative to such a tile: rows 4*(lane/16) + (lane%16)/4 (k-slots
// 0..3; +kRmHighRows for 4..7), d from 32*(lane%4) + 8*j, at the swizzled chunk position.
__device__ inline uint32_t tr_lane_off(int lane, int j) {
  const int lg = lane >> 4, lr = lane & 15;
  return rm_block_off(lg) + 256u * (uint32_t)(lr >> 2) + 16u * (uint32_t)((4 * (lr & 3) + j) ^ (lr >> 2));
}

// Transposed operands (V^T in the forward, K^T in the dQ product) of all 8 d-tiles straight from a
// row-major tile of 32 key rows in LDS with the transposing read ds_read_b64_tr_b16.  Within each
// 16-lane group that read hands lane i, element j, element i%4 of the 8 bytes that lane 4j + i/4
// addressed.  The caller passes a[j] = tile + tr_lane_off(lane, j) (d-tiles 2j and 2j+1, k-slots
// 0..3); +8 selects the odd d-tile, +kRmHighRows (4128) the k-slots 4..7 (tile rows 16..31).  Result vt[dt],
// slot k of lane l: row[key slot 16*(k/4) + 4*(l/16) + k%4][d = 32*((l%16)/4) + 4*dt + l%4], so
// accumulator register r of d-tile dt in lane l holds d = 32*(l/16) + 4*dt + r.  One statement,
// ending in its own wait (direct-to-LDS loads in flight must not make it wait for them).
static_assert(kRmHighRows == 4128, "the read offsets below are kRmHighRows and kRmHighRows + 8");
__device__ inline void read_vt_tr(bf16x8 (&vt)[8], const uint32_t (&a)[4]) {
  uint64_t x[16];
  asm volatile(
      "ds_read_b64_tr_b16 %0, %16\n"
      "ds_read_b64_tr_b16 %1, %16 offset:4128\n"
      "ds_read_b64_tr_b16 %2, %16 offset:8\n"
      "ds_read_b64_tr_b16 %3, %16 offset:4136\n"
      "ds_read_b64_tr_b16 %4, %17\n"
      "ds_read_b64_tr_b16 %5, %17 offset:4128\n"
      "ds_read_b64_tr_b16 %6, %17 offset:8\n"
      "ds_read_b64_tr_b16 %7, %17 offset:4136\n"
      "ds_read_b64_tr_b16 %8, %18\n"
      "ds_read_b64_tr_b16 %9, %18 offset:4128\n"
      "ds_read_b64_tr_b16 %10, %18 offset:8\n"
      "ds_read_b64_tr_b16 %11, %18 offset:4136\n"
      "ds_read_b64_tr_b16 %12, %19\n"
      "ds_read_b64_tr_b16 %13, %19 offset:4128\n"
      "ds_read_b64_tr_b16 %14, %19 offset:8\n"
      "ds_read_b64_tr_b16 %15, %19 offset:4136\n"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(x[0]), "=&v"(x[1]), "=&v"(x[2]), "=&v"(x[3]), "=&v"(x[4]), "=&v"(x[5]), "=&v"(x[6]), "=&v"(x[7]),
        "=&v"(x[8]), "=&v"(x[9]), "=&v"(x[10]), "=&v"(x[11]), "=&v"(x[12]), "=&v"(x[13]), "=&v"(x[14]),
        "=&v"(x[15])
      : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]));
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) {
    const uint64_t lo = x[2 * dt], hi = x[2 * dt + 1];
    vt[dt] = as_bf16x8(u32x4{(uint32_t)lo, (uint32_t)(lo >> 32), (uint32_t)hi, (uint32_t)(hi >> 32)});
  }
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
