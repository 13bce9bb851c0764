// Backward of the continuation block's attention under its sparse views and the
// full cache (Alg. 1 steps 3-5: the drafter's losses reach the block's queries
// and, through the cache rows the block itself wrote, its keys and values; the
// prefix cache carries no gradient).
//
// For one branch (a view or the full cache) with softmax weights
// P[r][t] = exp(scale * q_r . k_t - lse_r) over the keys row r sees:
//   D_r     = <dO_r, O_r>                   (O_r the forward's fp32 output)
//   dS[r][t] = P[r][t] * (<dO_r, v_t> - D_r)
//   dQ_r    = scale * sum_t dS[r][t] k_t
//   dK_t    = scale * sum_r dS[r][t] q_r      (block rows t only)
//   dV_t    = sum_r P[r][t] dO_r             (block rows t only)
// and the branches add up.  The forward's log-sum-exp gives P directly, so no
// pass recomputes softmax statistics.
//
// dQ kernel.  Like the forward's block mode: a workgroup of 8 waves owns a
// share of one (sequence, KV head, row group) unit's key stream (the views'
// entry lists followed by the full branch's cache rows, cut into equal ranges
// at run time, when the list lengths are known); wave w owns the 32-row block
// 8*rg + w and every wave consumes every 32-key tile from a shared LDS ring
// filled by direct-to-LDS loads.  A tile carries K and V in the score operand
// layout and K a second time in the transposed layout of the dQ product, so
// every LDS read is a linear 1 KiB per instruction.  Per tile a wave runs
// three MFMA products (keys on the M side throughout):
//   S^T  [key][row] = K . Q^T          A = K tile,  B = Q^T   (registers)
//   dP^T [key][row] = V . dO^T         A = V tile,  B = dO^T  (registers)
//   dQ^T [d][row]  += K^T . dS^T       A = K^T,     B = dS^T  (P, dS never leave registers)
// dQ sums over the branches, so one accumulator serves the whole range.  Each
// workgroup's partial goes to a record; a merge kernel adds a unit's records
// in workgroup order, so the result does not depend on scheduling.  The
// workgroup holding a branch's first entry also publishes each row's (lse, D)
// for dK/dV.
//
// dK/dV kernel.  One workgroup of 8 waves per (sequence, KV head, branch), two
// groups of 4 taking alternate row tiles; wave w of a group owns 16 block
// keys, and the branch's query rows stream through a direct-to-LDS ring in
// 32-row tiles (Q and dO, each in the A-operand and the transposed layout).
// Per tile a wave runs
//   S  [row][key] = Q . K_blk^T        dP [row][key] = dO . V_blk^T
//   dV^T [d][key] += dO^T . P          dK^T [d][key] += Q^T . dS
// (P and dS as bf16 pairs hi + lo).  The branches' partials meet in records
// that a merge kernel sums in branch order.

#include "bd_common.hpp"
#include "bd_kernels.hpp"
#include "attn_tile.hpp"

namespace bd {
namespace {

constexpr int kTile = 32;                          // keys per tile
constexpr float kLog2e = 1.4426950408889634f;
constexpr int64_t kTargetBlocks = 256;             // one workgroup per CU

// ---- dQ kernel ----------------------------------------------------------------
constexpr int kQWaves = 8;
constexpr int kQThreads = kQWaves * kWave;
constexpr int kQRing = 5;                          // tile slots; kQRing-1 tiles in flight
constexpr int kQLoads = 24;                        // 16-byte loads per lane per tile (3 per wave)
constexpr int kQTileBytes = 16384 + kRmTileBytes; // K and V in the score layout, then K row-major
constexpr int kQSlotCap = kMaxSplitKeys + kQRing * kTile;
constexpr int kRecFloats = 2 * 16 * kD;            // one wave's dQ partial: 32 rows x 128

struct DqSmem {
  alignas(16) int32_t roff[kQSlotCap];
  alignas(16) int32_t tpos[kQSlotCap];
  alignas(16) uint8_t ring[kQRing][kQTileBytes];
};

// Tile load q of a lane (0..23).  q < 8: K, score layout (key sub-tile q/4 -> rows 16*(q/4) + lane%16,
// 16 bytes at d = 32*(lane/16) + 8*(q%4)); 8 <= q < 16: V, same layout; 16 <= q < 24: K again, as a
// row-major tile for the transposing reads of the dQ product (rm_row, rm_chunk).
__device__ inline int load_row_in_tile(int q, int lane) {
  const int lr = lane & 15;
  return q < 16 ? 16 * ((q & 7) >> 2) + lr : rm_row(q - 16, lane);
}
__device__ inline void dq_dma_load(const KvView& kv, uint32_t r, uint32_t max_roff, int q, uint8_t* dst, int lane) {
  const int lg = lane >> 4;
  const uint32_t ro = r < max_roff ? r : max_roff;
  const uint64_t base = (uint64_t)ro << 3;
  if (q < 8) dma16(kv.k + base + 32 * lg + 8 * (q & 3), dst + q * 1024);
  else if (q < 16) dma16(kv.v + base + 32 * lg + 8 * (q & 3), dst + q * 1024);
  else dma16(kv.k + base + 8 * rm_chunk(lane), dst + 16384 + rm_block_off(q - 16));
}

// Eight 1 KiB pieces of a tile (loads q0 .. q0+7) into registers, with their wait.
__device__ inline void read8(u32x4 (&x)[8], uint32_t a) {
  asm volatile(
      "ds_read_b128 %0, %8\n"
      "ds_read_b128 %1, %8 offset:1024\n"
      "ds_read_b128 %2, %8 offset:2048\n"
      "ds_read_b128 %3, %8 offset:3072\n"
      "ds_read_b128 %4, %8 offset:4096\n"
      "ds_read_b128 %5, %8 offset:5120\n"
      "ds_read_b128 %6, %8 offset:6144\n"
      "ds_read_b128 %7, %8 offset:7168\n"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(x[0]), "=&v"(x[1]), "=&v"(x[2]), "=&v"(x[3]), "=&v"(x[4]), "=&v"(x[5]), "=&v"(x[6]), "=&v"(x[7])
      : "v"(a));
}
// K pieces (score layout), the tile's key positions and the row offsets of this wave's next loads.
__device__ inline void read8_pos_rows(u32x4 (&x)[8], u32x4 (&tp)[2], uint32_t (&r)[3], uint32_t a, uint32_t ap,
                                      uint32_t a0, uint32_t a1, uint32_t a2) {
  asm volatile(
      "ds_read_b128 %0, %13\n"
      "ds_read_b128 %1, %13 offset:1024\n"
      "ds_read_b128 %2, %13 offset:2048\n"
      "ds_read_b128 %3, %13 offset:3072\n"
      "ds_read_b128 %4, %13 offset:4096\n"
      "ds_read_b128 %5, %13 offset:5120\n"
      "ds_read_b128 %6, %13 offset:6144\n"
      "ds_read_b128 %7, %13 offset:7168\n"
      "ds_read_b128 %8, %14\n"
      "ds_read_b128 %9, %14 offset:64\n"
      "ds_read_b32 %10, %15\n"
      "ds_read_b32 %11, %16\n"
      "ds_read_b32 %12, %17\n"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(x[0]), "=&v"(x[1]), "=&v"(x[2]), "=&v"(x[3]), "=&v"(x[4]), "=&v"(x[5]), "=&v"(x[6]), "=&v"(x[7]),
        "=&v"(tp[0]), "=&v"(tp[1]), "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2])
      : "v"(a), "v"(ap), "v"(a0), "v"(a1), "v"(a2));
}

// Per-wave row data of the dQ kernel: rows 16*nt + lane%16 of the wave's 32-row block.
struct DqRows {
  bf16x8 qop[2][4];   // Q^T operand (d slots 32*(lane/16) + 8*kk ..)
  bf16x8 dop[2][4];   // dO^T operand, same layout
  float lse2[2];      // log-sum-exp in log2 units (+inf: the row's weights are all zero)
  float Dr[2];        // <dO_r, O_r>
  int rowpos[2];
};

// One 32-key tile: dQ^T[nt][dt] += K^T . (P o (dP - D))^T.  `kreg` holds the K pieces (score layout)
// already read; the V and transposed-K pieces are read from the slot at `src`.  dS enters the product
// as a bf16 pair hi + lo (lo the rounded remainder): where a row's weight concentrates, dS terms of
// both signs nearly cancel in dQ and a single bf16 rounding of dS would dominate the result's error.
// ktr_off: this lane's read_vt_tr offsets of the tile's row-major K (16 KiB + tr_lane_off); dQ^T
// register r of d-tile dt then holds d = 32*(lane/16) + 4*dt + r.
template <class PosFn>
__device__ inline void dq_tile_step(f32x4 (&acc)[2][8], const DqRows& rw, const u32x4 (&kreg)[8], uint32_t src,
                                    const uint32_t (&ktr_off)[4], int lane, float scale_log2, bool dirty,
                                    PosFn pos_of) {
  f32x4 p[2][2];
#pragma unroll
  for (int sub = 0; sub < 2; ++sub)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      f32x4 a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < 4; ++j)
        a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kreg[4 * sub + j]), rw.qop[nt][j], a, 0, 0, 0);
      p[sub][nt] = a;
    }
  if (dirty) {
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int tpos = pos_of(i);
        if (!(tpos >= 0 && tpos <= rw.rowpos[nt])) p[i >> 2][nt][i & 3] = -INFINITY;
      }
  }
#pragma unroll
  for (int sub = 0; sub < 2; ++sub)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        p[sub][nt][e] = __builtin_amdgcn_exp2f(fmaf(p[sub][nt][e], scale_log2, -rw.lse2[nt]));

  u32x4 vreg[8];
  read8(vreg, src + 8 * 1024 + 16 * lane);
  bf16x8 dsop[2], dslo[2];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    f32x4 dp[2];
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      f32x4 a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < 4; ++j)
        a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vreg[4 * sub + j]), rw.dop[nt][j], a, 0, 0, 0);
      dp[sub] = a;
    }
    u32x4 w, wl;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int i0 = 2 * i, i1 = 2 * i + 1;
      const float d0 = p[i0 >> 2][nt][i0 & 3] * (dp[i0 >> 2][i0 & 3] - rw.Dr[nt]);
      const float d1 = p[i1 >> 2][nt][i1 & 3] * (dp[i1 >> 2][i1 & 3] - rw.Dr[nt]);
      w[i] = pack_bf16x2(d0, d1);
      wl[i] = pack_bf16x2(d0 - bf16_lo(w[i]), d1 - bf16_hi(w[i]));
    }
    dsop[nt] = as_bf16x8(w);
    dslo[nt] = as_bf16x8(wl);
  }

  bf16x8 kts[8];
  {
    const uint32_t a4[4] = {src + ktr_off[0], src + ktr_off[1], src + ktr_off[2], src + ktr_off[3]};
    read_vt_tr(kts, a4);
  }
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) {
    const bf16x8 a = kts[dt];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      acc[nt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, dsop[nt], acc[nt][dt], 0, 0, 0);
      acc[nt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, dslo[nt], acc[nt][dt], 0, 0, 0);
    }
  }
}

// Every kernel argument line requested at entry, so the arguments cost one memory round trip (the
// compiler would otherwise fetch each where it is first used).  The statements touch no memory and
// return 0, which the caller adds to its block index.
__device__ inline int fetch_bwd_args(const AttnBwdParams& p) {
  int z0, z1;
  asm("s_mov_b32 %0, 0" : "=s"(z0) : "s"(p.kv.k), "s"(p.kv.v), "s"(p.kv.seq_lens), "s"(p.kv.page_table),
      "s"(p.kv.stride_seq), "s"(p.kv.stride_head), "s"(p.kv.stride_tok), "s"(p.kv.stride_page), "s"(p.q),
      "s"(p.o32_g), "s"(p.lse_g), "s"(p.dout_g), "s"(p.o32_f), "s"(p.lse_f), "s"(p.dout_f));
  asm("s_mov_b32 %0, 0" : "=s"(z1) : "s"(z0), "s"(p.idx), "s"(p.nsel), "s"(p.ld_idx), "s"(p.S), "s"(p.R),
      "s"(p.nW), "s"(p.nkt), "s"(p.scale_log2), "s"(p.max_roff), "s"(p.dq), "s"(p.part_q), "s"(p.rstats),
      "s"(p.R_pad), "s"(p.counters));
  return z1;
}
// The dK/dV kernel's arguments, requested at entry the same way (fetched where first used they took
// four round trips before its first data load).
__device__ inline int fetch_dkv_args(const AttnBwdParams& p) {
  int z0, z1, z2;
  asm("s_mov_b32 %0, 0" : "=s"(z0) : "s"(p.kv.k), "s"(p.kv.v), "s"(p.kv.seq_lens), "s"(p.kv.page_table),
      "s"(p.kv.stride_seq), "s"(p.kv.stride_head), "s"(p.kv.stride_tok), "s"(p.kv.stride_page), "s"(p.kv.max_seq_len),
      "s"(p.kv.page_size), "s"(p.kv.max_pages_per_seq), "s"(p.kv.num_pages));
  asm("s_mov_b32 %0, 0" : "=s"(z1) : "s"(z0), "s"(p.q), "s"(p.o32_g), "s"(p.lse_g), "s"(p.dout_g), "s"(p.o32_f),
      "s"(p.lse_f), "s"(p.dout_f), "s"(p.idx), "s"(p.nsel), "s"(p.ld_idx), "s"(p.S), "s"(p.Hkv), "s"(p.Hq));
  asm("s_mov_b32 %0, 0" : "=s"(z2) : "s"(z1), "s"(p.G), "s"(p.C), "s"(p.V), "s"(p.R), "s"(p.n_rb), "s"(p.nbr),
      "s"(p.nkt), "s"(p.scale), "s"(p.scale_log2), "s"(p.inv_G), "s"(p.max_roff), "s"(p.dk), "s"(p.dv),
      "s"(p.part_kv), "s"(p.rstats), "s"(p.R_pad));
  return z2;
}
// Workgroup barrier for LDS traffic: waits for this wave's LDS operations only, not for its global
// loads in flight (which a __syncthreads fence would wait for).
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// The dQ kernel's cut of a unit's key stream (StreamCut): equal shares starting on whole tiles.
// Weighting gathered entries more, as the forward does, was slower here (163 vs 144 us; 178 vs
// 137 us with all pieces of a range in one slot table): the gathered tiles of the views, each row
// a separate 256-byte read of three tile pieces, slow down as more workgroups stream them at once.
constexpr int kQWGather = 1, kQWFull = 1;
using DqCut = StreamCut<kQWGather, kQWFull, kTile>;

template <bool PAGED>
__global__ __launch_bounds__(kQThreads) void dq_kernel(AttnBwdParams p) {
  __shared__ DqSmem sm;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lg = lane >> 4, lr = lane & 15;

  // ---- unit (sequence, KV head, row group) and this workgroup's share w of the unit's key stream
  const int bid = xcd_remap(blockIdx.x + fetch_bwd_args(p), gridDim.x);
  const int w = bid % p.nW;
  const int unit = bid / p.nW;
  const int rg = unit % p.n_rg;
  const int pair = unit / p.n_rg;
  const int g = pair % p.Hkv, s = pair / p.Hkv;
  const int rb = rg * kQWaves + wave;
  const bool has_rows = rb < p.n_rb;
  const int L = seq_len(p.kv, s);

  // The key stream of a unit is the views' entry lists followed by the full branch's cache rows;
  // its actual length is known only here (nsel lives on the device), so the unit's nW workgroups
  // cut it into equal weighted shares at run time (DqCut).  A range crossing a branch boundary runs
  // one piece per branch (each with the branch's dO, D and lse rows).
  auto branch_len = [&](int b) -> int {
    if (b < p.V) {
      const int n = p.nsel[b * p.S + s];
      return n < 0 ? 0 : (n > p.ld_idx ? p.ld_idx : n);
    }
    return L;
  };
  int total = 0, vt = 0;
  for (int b = 0; b < p.nbr; ++b) {
    const int n = branch_len(b);
    total += n;
    if (b < p.V) vt += n;
  }
  const DqCut cut(vt, total, p.nW);
  const int r0 = cut.start_of(w), r1 = cut.start_of(w + 1);

  // ---- this wave's rows: Q once; dO, lse and D = <dO, O> per branch
  const int64_t branch_rows = (int64_t)p.S * p.C * p.Hq;
  DqRows rw;
  int64_t orow[2];
  bool rvalid[2];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    const int n = rb * 32 + 16 * nt + lr;
    rvalid[nt] = has_rows && n < p.R;
    const int j = rvalid[nt] ? n / p.G : 0;
    const int h = g * p.G + (rvalid[nt] ? n % p.G : 0);
    orow[nt] = ((int64_t)s * p.C + j) * p.Hq + h;
    rw.rowpos[nt] = rvalid[nt] ? L - p.C + j : 0x7FFFFFFF;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      rw.qop[nt][kk] = as_bf16x8(rvalid[nt] ? load16(p.q + orow[nt] * kD + 32 * lg + 8 * kk) : u32x4{0u, 0u, 0u, 0u});
  }
  // A branch's rows: the loads are issued before the piece's slot table is filled (its idx loads
  // then share their round trip), the sums D = <dO, O> taken after it.
  struct BranchRaw {
    u32x4 dv[2][4];
    f32x4 o[2][4][2];
    float lse[2];
  };
  auto issue_branch_rows = [&](int b, BranchRaw& x) {
    const bool gb = b < p.V;
    const float* outb = gb ? p.o32_g + (int64_t)b * branch_rows * kD : p.o32_f;
    const uint16_t* doutb = gb ? p.dout_g + (int64_t)b * branch_rows * kD : p.dout_f;
    const float* lseb = gb ? p.lse_g + (int64_t)b * branch_rows : p.lse_f;
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int64_t off = orow[nt] * kD + 32 * lg + 8 * kk;
        x.dv[nt][kk] = rvalid[nt] ? load16(doutb + off) : u32x4{0u, 0u, 0u, 0u};
        x.o[nt][kk][0] = rvalid[nt] ? *reinterpret_cast<const f32x4*>(outb + off) : f32x4{0.f, 0.f, 0.f, 0.f};
        x.o[nt][kk][1] = rvalid[nt] ? *reinterpret_cast<const f32x4*>(outb + off + 4) : f32x4{0.f, 0.f, 0.f, 0.f};
      }
      x.lse[nt] = rvalid[nt] ? lseb[orow[nt]] : INFINITY;
    }
  };
  auto finish_branch_rows = [&](const BranchRaw& x) {
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      float dsum = 0.f;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const u32x4 dv = x.dv[nt][kk];
        const f32x4 o0 = x.o[nt][kk][0], o1 = x.o[nt][kk][1];
        rw.dop[nt][kk] = as_bf16x8(dv);
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          dsum += bf16_lo(dv[e]) * o0[2 * e] + bf16_hi(dv[e]) * o0[2 * e + 1];
          dsum += bf16_lo(dv[e + 2]) * o1[2 * e] + bf16_hi(dv[e + 2]) * o1[2 * e + 1];
        }
      }
      rw.Dr[nt] = sum_xor32(sum_xor16(dsum));
      const float l2 = x.lse[nt] * kLog2e;
      rw.lse2[nt] = l2 == -INFINITY ? INFINITY : l2;   // a row that saw no key has all-zero weights
    }
  };

  const int minpos = L - p.C + (rb * 32) / p.G;   // earliest row position of this wave
  f32x4 acc[2][8];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt)
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) acc[nt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // ---- the three loads of every tile that this wave issues
  const int q0 = 3 * wave;
  const int rit0 = load_row_in_tile(q0, lane), rit1 = load_row_in_tile(q0 + 1, lane),
            rit2 = load_row_in_tile(q0 + 2, lane);
  uint32_t ktr_off[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) ktr_off[j] = 16384u + tr_lane_off(lane, j);
  const uint32_t roff_lds = lds_addr(sm.roff), tpos_lds = lds_addr(sm.tpos);
  const uint32_t ring_lds = lds_addr(sm.ring[0]);
  auto issue = [&](int tile, const uint32_t (&r)[3]) {
    uint8_t* dst = sm.ring[tile % kQRing];
    dq_dma_load(p.kv, r[0], p.max_roff, q0, dst, lane);
    dq_dma_load(p.kv, r[1], p.max_roff, q0 + 1, dst, lane);
    dq_dma_load(p.kv, r[2], p.max_roff, q0 + 2, dst, lane);
  };

  // entries e_begin .. e_end-1 of one branch through the slot table (a piece never exceeds it)
  auto stream = [&](int e_begin, int e_end) {
    const int ntiles = (e_end - e_begin + kTile - 1) / kTile;
    for (int t = 0; t < kQRing - 1; ++t) {
      uint32_t r[3];
      asm volatile(
          "ds_read_b32 %0, %3\n"
          "ds_read_b32 %1, %4\n"
          "ds_read_b32 %2, %5\n"
          "s_waitcnt lgkmcnt(0)"
          : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2])
          : "v"(roff_lds + 4 * (kTile * t + rit0)), "v"(roff_lds + 4 * (kTile * t + rit1)),
            "v"(roff_lds + 4 * (kTile * t + rit2)));
      issue(t, r);
    }
    for (int t = 0; t < ntiles; ++t) {
      // this wave's loads of tile t are older than the kQRing-2 tiles issued after it
      asm volatile("s_waitcnt vmcnt(9)\n\ts_barrier" ::: "memory");
      static_assert(3 * (kQRing - 2) == 9, "wait count follows the ring depth");
      const int nxt = t + kQRing - 1;
      const uint32_t src = ring_lds + (uint32_t)(t % kQRing) * kQTileBytes;
      u32x4 kreg[8];
      uint32_t r[3];
      u32x4 tp[2];
      const int next0 = kTile * nxt;
      read8_pos_rows(kreg, tp, r, src + 16 * lane, tpos_lds + 4 * (kTile * t + 4 * lg),
                     roff_lds + 4 * (next0 + rit0), roff_lds + 4 * (next0 + rit1), roff_lds + 4 * (next0 + rit2));
      bool bad = false;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int tq = (int)tp[i >> 2][i & 3];
        bad |= tq < 0 || tq > minpos;
      }
      const bool dirty = __builtin_amdgcn_ballot_w64(bad) != 0;
      issue(nxt, r);
      if (has_rows)
        dq_tile_step(acc, rw, kreg, src, ktr_off, lane, p.scale_log2, dirty,
                     [&](int i) { return (int)tp[i >> 2][i & 3]; });
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // padding loads land before the ring is reused
  };

  int off = 0;
  for (int b = 0; b < p.nbr; ++b) {
    const int n = branch_len(b);
    const int lo = r0 > off ? r0 : off, hi = r1 < off + n ? r1 : off + n;
    off += n;
    if (lo >= hi) continue;
    const int e0 = lo - (off - n), e1 = hi - (off - n);
    BranchRaw raw;
    issue_branch_rows(b, raw);
    const int32_t* idx_row = b < p.V ? p.idx + (((int64_t)b * p.S + s) * p.Hkv + g) * p.ld_idx : nullptr;
    const int nslots = ((e1 - e0 + kTile - 1) / kTile + kQRing) * kTile;
    // these barriers wait for LDS traffic alone (a __syncthreads fence would wait for the rows too)
    lds_barrier();                                // the previous piece's slot table and ring are free
    fill_slot_table<PAGED, kQThreads, kQSlotCap>(p.kv, s, g, L, idx_row, e0, e1, nslots, sm.roff, sm.tpos, tid);
    lds_barrier();
    finish_branch_rows(raw);
    if (e0 == 0 && p.rstats && lg == 0) {         // the branch's first workgroup publishes the row stats
      float* rs = p.rstats + (((int64_t)b * p.S * p.Hkv + pair) * p.R_pad + rb * 32) * 2;
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
        if (rvalid[nt]) *reinterpret_cast<float2*>(rs + 2 * (16 * nt + lr)) = float2{rw.lse2[nt], rw.Dr[nt]};
    }
    stream(e0, e1);
  }

  // ---- dQ rows 16*nt + lane%16; register r of d-tile dt holds d = 32*(lane/16) + 4*dt + r
  auto write_rows = [&](const f32x4 (&o)[2][8]) {
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      if (!rvalid[nt]) continue;
      float* drow = p.dq + orow[nt] * kD + 32 * lg;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) *reinterpret_cast<f32x4*>(drow + 4 * dt) = o[nt][dt] * p.scale;
    }
  };
  if (p.nW == 1) {
    if (has_rows) write_rows(acc);
    return;
  }

  // ---- publish this wave's partial as record w of its row block: chunk (nt, dt) x lane float4s;
  // bwd_merge_kernel, launched after the dK/dV kernel, sums them
  if (has_rows) {
    const __amdgpu_buffer_rsrc_t urec =
        make_rsrc(p.part_q + ((int64_t)unit * kQWaves + wave) * p.nW * kRecFloats, (uint32_t)(p.nW * kRecFloats * 4));
    const uint32_t rec = (uint32_t)w * kRecFloats * 4;
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) store16_coherent(urec, rec + 16 * ((nt * 8 + dt) * kWave + lane), acc[nt][dt]);
  }
}

// Sum of the dQ partials: one wave per (unit, row block, row tile nt, half dh of the d-tiles) adds
// the nW workgroups' records in workgroup order, so the result does not depend on scheduling.  A
// separate launch spreads it over the chip: summed by the unit's last workgroup, 8 records of
// 128 KiB went into one CU (15 us at one CU's bandwidth).  Every load of a batch of kQMBatch
// records is issued before any is added.  Block `id` of the merge kernel's dQ part.
constexpr int kQMBatch = 8;
__device__ inline void dq_merge_block(const AttnBwdParams& p, int id) {
  const int lane = threadIdx.x, lg = lane >> 4, lr = lane & 15;
  const int dh = id & 1, nt = (id >> 1) & 1;
  id >>= 2;
  const int wave = id % kQWaves, unit = id / kQWaves;
  const int rg = unit % p.n_rg, pair = unit / p.n_rg;
  const int g = pair % p.Hkv, s = pair / p.Hkv;
  const int rb = rg * kQWaves + wave;
  if (rb >= p.n_rb) return;
  const int n = rb * 32 + 16 * nt + lr;
  const __amdgpu_buffer_rsrc_t urec =
      make_rsrc(p.part_q + ((int64_t)unit * kQWaves + wave) * p.nW * kRecFloats, (uint32_t)(p.nW * kRecFloats * 4));
  f32x4 o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int k = 0; k < p.nW; k += kQMBatch) {
    f32x4 x[kQMBatch][4];
#pragma unroll
    for (int kk = 0; kk < kQMBatch; ++kk)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        x[kk][i] = k + kk < p.nW ? load16_coherent(urec, (uint32_t)(k + kk) * kRecFloats * 4 +
                                                             16 * ((nt * 8 + 4 * dh + i) * kWave + lane))
                                 : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < kQMBatch; ++kk)
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] += x[kk][i];
  }
  if (n >= p.R) return;
  // register r of d-tile dt = 4*dh + i holds d = 32*lg + 4*dt + r
  const int j = n / p.G, h = g * p.G + n % p.G;
  float* drow = p.dq + (((int64_t)s * p.C + j) * p.Hq + h) * kD + 32 * lg + 16 * dh;
#pragma unroll
  for (int i = 0; i < 4; ++i) *reinterpret_cast<f32x4*>(drow + 4 * i) = o[i] * p.scale;
}

// ---- dK/dV kernel ---------------------------------------------------------------
// One workgroup of 8 waves per (sequence, KV head, branch, pass of 64 block keys) in two groups of
// 4: wave w of a group owns the 16 block keys of key tile 4*pass + w, group 0 takes the
// even 32-row tiles of the branch's query rows and group 1 the odd ones, and the groups' partial
// sums are added in LDS at the end (two waves per SIMD: one wave's MFMA chains and LDS reads
// overlap the other's).  The row tiles stream through an LDS ring, each tile carrying Q and dO
// twice: in the A-operand layout of the S and dP products and in the transposed layout of the dK
// and dV products, so every LDS read is linear.
constexpr int kKGroupWaves = 4;
constexpr int kKWaves = 2 * kKGroupWaves;
constexpr int kKThreads = kKWaves * kWave;
constexpr int kKRing = 4;                          // row-tile slots: two per group, one in flight
constexpr int kKLoads = 32;                        // 1 KiB pieces per row tile (8 per wave)
constexpr int kKStatBytes = 32 * 8;                // the tile's rows' (lse2, D) pairs (64 bytes per wave)
constexpr int kKTileBytes = kKLoads * 1024 + kKStatBytes;

struct DkvSmem {
  alignas(16) uint8_t ring[kKRing][kKTileBytes];
  int32_t cnt[kMaxBwdBlock];                       // occurrences of block key c in the branch's key list
};

// Piece q (0..31) of a row tile for this lane: 0..7 Q in the A layout (rows 16*(q/4) + lane%16,
// 16 bytes at d = 32*(lane/16) + 8*(q%4)), 8..15 Q transposed (rows 16*((q-8)/4) + 4*(lane/16) +
// (q-8)%4, 16 bytes at d = 8*(lane%16)), 16..31 the same two for dO.
__device__ inline void row_piece(int q, int lane, int& r, int& d) {
  const int lg = lane >> 4, lr = lane & 15, x = q & 7;
  if ((q & 8) == 0) { r = 16 * (x >> 2) + lr; d = 32 * lg + 8 * (x & 3); }
  else { r = 16 * (x >> 2) + 4 * lg + (x & 3); d = 8 * lr; }
}

template <bool PAGED>
__global__ __launch_bounds__(kKThreads) void dkv_kernel(AttnBwdParams p) {
  __shared__ DkvSmem sm;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave / kKGroupWaves, wk = wave % kKGroupWaves;
  const int lg = lane >> 4, lr = lane & 15;
  const int bid = xcd_remap(blockIdx.x + fetch_dkv_args(p), gridDim.x);
  const int br = bid % p.nbr;
  const int npass = (p.nkt + kKGroupWaves - 1) / kKGroupWaves;
  const int kpass = (bid / p.nbr) % npass;       // the block keys' pass: key tiles 4*kpass .. +3
  const int pair = bid / p.nbr / npass;          // s * Hkv + g
  const int g = pair % p.Hkv, s = pair / p.Hkv;
  const bool gather = br < p.V;
  const int L = seq_len(p.kv, s);
  const int C = p.C, t0 = L - C;                 // block row c sits at position t0 + c

  // ---- key multiplicities of the branch (all idx loads of a round issued before any atomic)
  for (int c = tid; c < C; c += kKThreads) sm.cnt[c] = (!gather && t0 + c >= 0) ? 1 : 0;
  __syncthreads();
  if (gather) {
    const int32_t* idx_row = p.idx + (((int64_t)br * p.S + s) * p.Hkv + g) * p.ld_idx;
    int n = p.nsel[br * p.S + s];
    n = n < 0 ? 0 : (n > p.ld_idx ? p.ld_idx : n);
    constexpr int kPer = 8;
    for (int e0 = 0; e0 < n; e0 += kPer * kKThreads) {
      int tv[kPer];
#pragma unroll
      for (int k = 0; k < kPer; ++k) {
        const int e = e0 + tid + k * kKThreads;
        tv[k] = e < n ? idx_row[e] : -1;
      }
#pragma unroll
      for (int k = 0; k < kPer; ++k)
        if (tv[k] >= 0 && tv[k] < L && tv[k] >= t0) atomicAdd(&sm.cnt[tv[k] - t0], 1);
    }
    __syncthreads();
  }

  const int64_t branch_rows = (int64_t)p.S * C * p.Hq;
  const uint16_t* doutb = gather ? p.dout_g + (int64_t)br * branch_rows * kD : p.dout_f;
  // (lse2, D) of the branch's rows of this (s, g), published by the dQ kernel, rows padded to R_pad
  const float* stats = p.rstats + ((int64_t)br * p.S * p.Hkv + pair) * p.R_pad * 2;
  const int nrt = (p.R + 31) / 32;
  const int nkt = (C + 15) / 16;
  auto row_off = [&](int n) -> int64_t {         // rows past R read row 0 (their weights are zero)
    const int nn = n < p.R ? n : 0;
    const int j = div_small(nn, p.G, p.inv_G);
    return ((int64_t)s * C + j) * p.Hq + g * p.G + (nn - j * p.G);
  };
  // this wave's 8 pieces of its group's row tiles
  int prow[8], pd[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) row_piece(8 * wk + k, lane, prow[k], pd[k]);
  const uint16_t* psrc = wk < 2 ? p.q : doutb;
  // step i: group g works on row tile 2i + g in ring slot g + 2*(i % 2)
  const int nit = (nrt + 1) / 2;
  auto slot_of = [&](int i) { return grp + 2 * (i & 1); };
  // 9 loads per wave and tile: its 8 pieces, and 64 bytes of the tile's row stats (lanes 0..3)
  auto issue = [&](int i) {
    const int rt = 2 * i + grp;
    uint8_t* dst = sm.ring[slot_of(i)];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int n = rt < nrt ? 32 * rt + prow[k] : 0;   // a padding tile re-reads row 0
      dma16(psrc + row_off(n) * kD + pd[k], dst + (8 * wk + k) * 1024);
    }
    const int srt = rt < nrt ? rt : 0;
    if (lane < 4)
      dma16(reinterpret_cast<const uint16_t*>(stats + srt * 64 + 16 * wk) + 8 * lane,
            dst + kKLoads * 1024 + 64 * wk);
  };
  const uint32_t ring_lds = lds_addr(sm.ring[0]);
  const __amdgpu_buffer_rsrc_t rrec =
      make_rsrc(p.part_kv + (int64_t)pair * p.nbr * C * 2 * kD, (uint32_t)((int64_t)p.nbr * C * 2 * kD * 4));
  const bool direct = p.nbr == 1;

  {
    const int kt0 = kKGroupWaves * kpass;
    const int kt = kt0 + wk;
    const int c = 16 * kt + lr;                  // this lane's key
    const bool kvalid = kt < nkt && c < C && t0 + c >= 0;
    const int mult = kvalid ? sm.cnt[c] : 0;
    // B operands K_blk^T and V_blk^T: lane l feeds key l%16 with d slots 32*(l/16) + 8*j ..
    bf16x8 kop[4], vop[4];
    {
      int64_t o = -1;
      if (mult > 0) o = row_offset<PAGED>(p.kv, s, g, t0 + c);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        kop[j] = as_bf16x8(o >= 0 ? load16(p.kv.k + o + 32 * lg + 8 * j) : u32x4{0u, 0u, 0u, 0u});
        vop[j] = as_bf16x8(o >= 0 ? load16(p.kv.v + o + 32 * lg + 8 * j) : u32x4{0u, 0u, 0u, 0u});
      }
    }
    const bool active = __builtin_amdgcn_ballot_w64(mult > 0) != 0;
    f32x4 dk[8], dv[8];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) dk[dt] = dv[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

    issue(0);
    for (int i = 0; i < nit; ++i) {
      // step i's tile landed for every wave of the group, and step i-1's slot is free: the next
      // tile of the group goes there while this one is computed
      asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
      if (i + 1 < nit) issue(i + 1);
      const int rt = 2 * i + grp;
      const uint32_t slot = ring_lds + (uint32_t)slot_of(i) * kKTileBytes;
      const uint32_t src = slot + 16 * lane;
      if (active && rt < nrt) {
        u32x4 qa[8], da[8];
        read8(qa, src);
        read8(da, src + 16 * 1024);
        // (lse2, D) of rows 16*sub + 4*lg + i: 32 contiguous bytes per sub
        f32x4 st[2][2];
        {
          const uint32_t a = slot + kKLoads * 1024 + 32 * lg;
          asm volatile(
              "ds_read_b128 %0, %4\n"
              "ds_read_b128 %1, %4 offset:16\n"
              "ds_read_b128 %2, %4 offset:128\n"
              "ds_read_b128 %3, %4 offset:144\n"
              "s_waitcnt lgkmcnt(0)"
              : "=&v"(st[0][0]), "=&v"(st[0][1]), "=&v"(st[1][0]), "=&v"(st[1][1])
              : "v"(a));
        }
        float l2[2][4], dd[2][4];
#pragma unroll
        for (int sub = 0; sub < 2; ++sub)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            l2[sub][i] = st[sub][i >> 1][2 * (i & 1)];
            dd[sub][i] = st[sub][i >> 1][2 * (i & 1) + 1];
          }
        // S [row][key] = Q . K_blk^T and dP [row][key] = dO . V_blk^T: lane l holds rows
        // 16*sub + 4*lg + i of key l%16
        f32x4 sp[2], dp[2];
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
          f32x4 x = {0.f, 0.f, 0.f, 0.f}, y = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            x = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(qa[4 * sub + j]), kop[j], x, 0, 0, 0);
            y = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(da[4 * sub + j]), vop[j], y, 0, 0, 0);
          }
          sp[sub] = x;
          dp[sub] = y;
        }
        u32x4 pw, dsw, pwl, dswl;
#pragma unroll
        for (int i2 = 0; i2 < 4; ++i2) {
          float pv[2], dsv[2];
#pragma unroll
          for (int e2 = 0; e2 < 2; ++e2) {
            const int slot = 2 * i2 + e2;                     // k-slot: row 16*(slot/4) + 4*lg + slot%4
            const int sub = slot >> 2, i = slot & 3;
            const int n = 32 * rt + 16 * sub + 4 * lg + i;
            const bool vis = mult > 0 && n < p.R && c <= div_small(n, p.G, p.inv_G);
            const float pr = vis ? __builtin_amdgcn_exp2f(fmaf(sp[sub][i], p.scale_log2, -l2[sub][i])) : 0.f;
            pv[e2] = pr;
            dsv[e2] = vis ? pr * (dp[sub][i] - dd[sub][i]) : 0.f;   // padding rows hold no stats
          }
          pw[i2] = pack_bf16x2(pv[0], pv[1]);
          dsw[i2] = pack_bf16x2(dsv[0], dsv[1]);
          pwl[i2] = pack_bf16x2(pv[0] - bf16_lo(pw[i2]), pv[1] - bf16_hi(pw[i2]));
          dswl[i2] = pack_bf16x2(dsv[0] - bf16_lo(dsw[i2]), dsv[1] - bf16_hi(dsw[i2]));
        }
        // transposed operands: register 4*h + i holds row 16*h + 4*lg + i, 16 bytes at d = 8*lr
        read8(qa, src + 8 * 1024);
        read8(da, src + 24 * 1024);
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
          const bf16x8 a_do = vt_operand(da, dt), a_q = vt_operand(qa, dt);
          dv[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_do, as_bf16x8(pw), dv[dt], 0, 0, 0);
          dv[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_do, as_bf16x8(pwl), dv[dt], 0, 0, 0);
          dk[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_q, as_bf16x8(dsw), dk[dt], 0, 0, 0);
          dk[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_q, as_bf16x8(dswl), dk[dt], 0, 0, 0);
        }
      }
    }
    // group 1 hands its partial sums to group 0 through the ring (16 KiB per wave)
    __syncthreads();                             // every ring read of the last step is done
    f32x4* red = reinterpret_cast<f32x4*>(sm.ring[0]) + wk * 16 * kWave + lane;
    if (grp == 1) {
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        red[dt * kWave] = dk[dt];
        red[(8 + dt) * kWave] = dv[dt];
      }
    }
    __syncthreads();
    if (grp == 0) {
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        dk[dt] += red[dt * kWave];
        dv[dt] += red[(8 + dt) * kWave];
      }
    }

    // key c: register i of d-tile dt holds d = 32*lg + 8*i + dt; a key listed m times counts m times
    if (grp == 0 && kt < nkt && c < C) {
      const float mk = (float)mult * (direct ? p.scale : 1.f), mv = (float)mult;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const f32x4 k0 = f32x4{dk[0][i], dk[1][i], dk[2][i], dk[3][i]} * mk;
        const f32x4 k1 = f32x4{dk[4][i], dk[5][i], dk[6][i], dk[7][i]} * mk;
        const f32x4 v0 = f32x4{dv[0][i], dv[1][i], dv[2][i], dv[3][i]} * mv;
        const f32x4 v1 = f32x4{dv[4][i], dv[5][i], dv[6][i], dv[7][i]} * mv;
        if (direct) {
          float* kr = p.dk + (((int64_t)s * C + c) * p.Hkv + g) * kD + 32 * lg + 8 * i;
          float* vr = p.dv + (((int64_t)s * C + c) * p.Hkv + g) * kD + 32 * lg + 8 * i;
          *reinterpret_cast<f32x4*>(kr) = k0;
          *reinterpret_cast<f32x4*>(kr + 4) = k1;
          *reinterpret_cast<f32x4*>(vr) = v0;
          *reinterpret_cast<f32x4*>(vr + 4) = v1;
        } else {
          const uint32_t ok = (uint32_t)((((int64_t)br * C + c) * 2 * kD + 32 * lg + 8 * i) * 4);
          const uint32_t ov = ok + (uint32_t)(kD * 4);
          store16_coherent(rrec, ok, k0);
          store16_coherent(rrec, ok + 16, k1);
          store16_coherent(rrec, ov, v0);
          store16_coherent(rrec, ov + 16, v1);
        }
      }
    }
  }
}

// Sum of the branches' dK/dV partials of every (sequence, KV head) in branch order, spread over the
// chip (the last of a pair's workgroups summing them alone was bound by one CU's bandwidth).  One
// thread per 16 bytes of a pair's record [C][dK | dV][128]; every load of a batch of 8 branches
// is issued before any is summed.  Block `id` of the merge kernel's dK/dV part.
__device__ inline int dkv_merge_blocks_per_pair(int C) { return (C * 2 * kD / 4 + kWave - 1) / kWave; }
__device__ inline void dkv_merge_block(const AttnBwdParams& p, int id) {
  const int chunks = p.C * 2 * kD / 4;           // float4s of one branch record
  const int per_pair = dkv_merge_blocks_per_pair(p.C);
  const int pair = id / per_pair;
  const int q = (id % per_pair) * kWave + threadIdx.x;
  if (q >= chunks) return;
  const int g = pair % p.Hkv, s = pair / p.Hkv;
  const __amdgpu_buffer_rsrc_t rrec =
      make_rsrc(p.part_kv + (int64_t)pair * p.nbr * p.C * 2 * kD, (uint32_t)((int64_t)p.nbr * p.C * 2 * kD * 4));
  constexpr int kBr = 8;
  f32x4 sum = {0.f, 0.f, 0.f, 0.f};
  for (int b0 = 0; b0 < p.nbr; b0 += kBr) {
    f32x4 x[kBr];
#pragma unroll
    for (int bb = 0; bb < kBr; ++bb)
      x[bb] = b0 + bb < p.nbr ? load16_coherent(rrec, (uint32_t)(((int64_t)(b0 + bb) * chunks + q) * 16))
                              : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int bb = 0; bb < kBr; ++bb) sum += x[bb];   // branch order (absent branches add 0)
  }
  const int fl = 4 * q;
  const int cc = fl / (2 * kD), rem = fl % (2 * kD);
  const bool isv = rem >= kD;
  const int d = isv ? rem - kD : rem;
  float* dst = (isv ? p.dv : p.dk) + (((int64_t)s * p.C + cc) * p.Hkv + g) * kD + d;
  *reinterpret_cast<f32x4*>(dst) = isv ? sum : sum * p.scale;
}

// Both sums in one launch of one-wave blocks: blocks [0, nq) sum the dQ partials, the rest the
// dK/dV partials.  The dK/dV kernel reads only what the dQ kernel publishes, so it runs before
// this merge and the two sums share the chip.
__global__ __launch_bounds__(kWave) void bwd_merge_kernel(AttnBwdParams p, int nq) {
  const int b = blockIdx.x;
  if (b < nq) dq_merge_block(p, b);
  else dkv_merge_block(p, b - nq);
}

}  // namespace

AttnBwdPlan plan_attn_bwd(int S, int Hkv, int Hq, int C, int num_views, int ld_idx, int max_L, bool with_full,
                          bool with_dkv) {
  AttnBwdPlan pl{};
  // counts held in int fields saturate at 2^30 (the caller rejects such shapes after planning)
  auto sat = [](int64_t x) { return x > (int64_t(1) << 30) ? (1 << 30) : (int)x; };
  const int G = Hq / Hkv;
  pl.R = sat((int64_t)C * G);
  pl.n_rb = (pl.R + 31) / 32;
  pl.n_rg = (pl.n_rb + kQWaves - 1) / kQWaves;
  pl.units = sat((int64_t)S * Hkv * pl.n_rg);
  pl.nbr = sat((int64_t)num_views + (with_full ? 1 : 0));
  pl.counter_bytes = BD_WS_COUNTER_BYTES;
  if (pl.nbr > 64) {                 // more branches than supported: the caller rejects the shape
    pl.ws_bytes = pl.counter_bytes;
    return pl;
  }
  pl.nkt = (C + 15) / 16;
  // workgroups per unit: enough to fill the CUs once, and enough that no range overflows the slot
  // table (a piece's range is at most kMaxSplitKeys entries)
  const int64_t stream_max = (int64_t)num_views * ld_idx + (with_full ? max_L : 0);
  int64_t nw = (kTargetBlocks + pl.units - 1) / pl.units;
  const int64_t nw_table = stream_cut_min_workgroups<kQWGather, kQWFull>(stream_max, kMaxSplitKeys);
  if (nw < nw_table) nw = nw_table;
  if (nw < 1) nw = 1;
  pl.nW = (int)nw;
  pl.nblk_q = sat((int64_t)pl.units * nw);
  // dK/dV workgroups: 64 keys each
  pl.nblk_kv = with_dkv ? sat((int64_t)S * Hkv * pl.nbr * ((pl.nkt + kKGroupWaves - 1) / kKGroupWaves)) : 0;
  pl.q_record_bytes = nw > 1 ? align256(sizeof(float) * kRecFloats * (size_t)pl.units * kQWaves * nw) : 0;
  pl.kv_record_bytes =
      with_dkv && pl.nbr > 1 ? align256(sizeof(float) * (size_t)S * Hkv * pl.nbr * C * 2 * kD) : 0;   // per key
  pl.R_pad = pl.n_rb * 32;
  pl.d_bytes = with_dkv ? align256(sizeof(float) * 2 * (size_t)pl.nbr * S * Hkv * pl.R_pad) : 0;
  pl.ws_bytes = pl.counter_bytes + pl.q_record_bytes + pl.kv_record_bytes + pl.d_bytes;
  return pl;
}

hipError_t launch_attn_bwd(const AttnBwdParams& p, const AttnBwdPlan& pl, bool paged, hipStream_t stream) {
  if (pl.nblk_q > 0) {
    if (paged) hipLaunchKernelGGL(dq_kernel<true>, dim3(pl.nblk_q), dim3(kQThreads), 0, stream, p);
    else hipLaunchKernelGGL(dq_kernel<false>, dim3(pl.nblk_q), dim3(kQThreads), 0, stream, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (pl.nblk_kv > 0) {
    if (paged) hipLaunchKernelGGL(dkv_kernel<true>, dim3(pl.nblk_kv), dim3(kKThreads), 0, stream, p);
    else hipLaunchKernelGGL(dkv_kernel<false>, dim3(pl.nblk_kv), dim3(kKThreads), 0, stream, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  // (unit, row block, row tile, d half) waves for dQ when the workgroups' partials need a sum;
  // (pair, 16-byte column block) waves for dK/dV when more than one branch contributes
  const int64_t nq = pl.nblk_q > 0 && pl.nW > 1 ? (int64_t)pl.units * kQWaves * 4 : 0;
  const int64_t nkv = pl.nblk_kv > 0 && pl.nbr > 1
                          ? (int64_t)p.S * p.Hkv * (((int64_t)p.C * 2 * kD / 4 + kWave - 1) / kWave)
                          : 0;
  if (nq + nkv == 0) return hipSuccess;
  hipLaunchKernelGGL(bwd_merge_kernel, dim3((unsigned)(nq + nkv)), dim3(kWave), 0, stream, p, (int)nq);
  return hipGetLastError();
}

}  // namespace bd
