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
// dQ kernel.  Like the forward's block mode: a workgroup of 8 waves owns one
// (branch, sequence, KV head, row group, key split); wave w owns the 32-row
// block 8*rg + w and every wave consumes every 32-key tile from a shared LDS
// ring filled by direct-to-LDS loads.  A tile carries K and V in the score
// operand layout and K a second time in the transposed layout of the dQ
// product, so every LDS read is a linear 1 KiB per instruction.  Per tile a
// wave runs three MFMA products (keys on the M side throughout):
//   S^T  [key][row] = K . Q^T          A = K tile,  B = Q^T   (registers)
//   dP^T [key][row] = V . dO^T         A = V tile,  B = dO^T  (registers)
//   dQ^T [d][row]  += K^T . dS^T       A = K^T,     B = dS^T  (P, dS never leave registers)
// Partial dQ of every (branch, split) goes to a record; the last workgroup of
// the (sequence, KV head, row group) adds them in (branch, split) order, so the
// result does not depend on which workgroup finishes when.
//
// dK/dV kernel.  One workgroup of 4 waves per (sequence, KV head, branch);
// wave w owns the 16 block keys of key tile w (then w+4, ...).  Row tiles of 32
// query rows are staged in padded row-major LDS (conflict-free for both the
// row-major and the transposed reads) and each wave runs, per row tile,
//   S  [row][key] = Q . K_blk^T        dP [row][key] = dO . V_blk^T
//   dV^T [d][key] += dO^T . P          dK^T [d][key] += Q^T . dS
// (P and dS again as bf16 pairs hi + lo).
// The branches' partials meet in records summed in branch order by the last.

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
constexpr int kQTileBytes = kQLoads * kWave * 16;  // 24 KiB
constexpr int kQSlotCap = kMaxSplitKeys + kQRing * kTile;
constexpr int kRecFloats = 2 * 16 * kD;            // one wave's dQ partial: 32 rows x 128

struct DqSmem {
  alignas(16) int32_t roff[kQSlotCap];
  alignas(16) int32_t tpos[kQSlotCap];
  alignas(16) uint8_t ring[kQRing][kQTileBytes];
  int32_t last;
};

// Tile load q of a lane (0..23).  q < 8: K, score layout (key sub-tile q/4 -> rows 16*(q/4) + lane%16,
// 16 bytes at d = 32*(lane/16) + 8*(q%4)); 8 <= q < 16: V, same layout; 16 <= q < 24: K, transposed
// layout (rows 16*((q-16)/4) + 4*(lane/16) + (q-16)%4, 16 bytes at d = 8*(lane%16)).
__device__ inline int load_row_in_tile(int q, int lane) {
  const int lg = lane >> 4, lr = lane & 15;
  return q < 16 ? 16 * ((q & 7) >> 2) + lr : 16 * ((q - 16) >> 2) + 4 * lg + ((q - 16) & 3);
}
__device__ inline void dq_dma_load(const KvView& kv, uint32_t r, uint32_t max_roff, int q, uint8_t* dst, int lane) {
  const int lg = lane >> 4, lr = lane & 15;
  const uint32_t ro = r < max_roff ? r : max_roff;
  const uint64_t base = (uint64_t)ro << 3;
  if (q < 8) dma16(kv.k + base + 32 * lg + 8 * (q & 3), dst + q * 1024);
  else if (q < 16) dma16(kv.v + base + 32 * lg + 8 * (q & 3), dst + q * 1024);
  else dma16(kv.k + base + 8 * lr, dst + q * 1024);
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
template <class PosFn>
__device__ inline void dq_tile_step(f32x4 (&acc)[2][8], const DqRows& rw, const u32x4 (&kreg)[8], uint32_t src,
                                    int lane, float scale_log2, bool dirty, PosFn pos_of) {
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

  u32x4 kt[8];
  read8(kt, src + 16 * 1024 + 16 * lane);
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) {
    const bf16x8 a = vt_operand(kt, dt);
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      acc[nt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, dsop[nt], acc[nt][dt], 0, 0, 0);
      acc[nt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, dslo[nt], acc[nt][dt], 0, 0, 0);
    }
  }
}

template <bool PAGED>
__global__ __launch_bounds__(kQThreads) void dq_kernel(AttnBwdParams p) {
  __shared__ DqSmem sm;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lg = lane >> 4, lr = lane & 15;

  // ---- (branch, sequence, head, row group, split) of this workgroup
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const bool gather = bid < p.nblk_g;
  const int local = gather ? bid : bid - p.nblk_g;
  const int nsplit = gather ? p.nsplit_g : p.nsplit_f;
  const int kps = gather ? p.kps_g : p.kps_f;
  const int rg = local % p.n_rg;
  const int rest = local / p.n_rg;
  const int split = rest % nsplit;
  const int pair = rest / nsplit;
  const int g = pair % p.Hkv;
  const int vs = pair / p.Hkv;                   // gather: view*S + s; full: s
  const int s = gather ? vs % p.S : vs;
  const int view = gather ? vs / p.S : 0;
  const int unit = (s * p.Hkv + g) * p.n_rg + rg;
  const int k_rec = gather ? view * p.nsplit_g + split : p.V * p.nsplit_g + split;
  const int rb = rg * kQWaves + wave;
  const bool has_rows = rb < p.n_rb;

  const int L = seq_len(p.kv, s);
  int n_keys;
  const int32_t* idx_row = nullptr;
  if (gather) {
    idx_row = p.idx + ((int64_t)vs * p.Hkv + g) * p.ld_idx;
    const int n = p.nsel[vs];
    n_keys = n < 0 ? 0 : (n > p.ld_idx ? p.ld_idx : n);
  } else {
    n_keys = L;
  }
  const int e_begin = split * kps;
  int e_end = e_begin + kps;
  if (e_end > n_keys) e_end = n_keys;
  const int ntiles = e_end > e_begin ? (e_end - e_begin + kTile - 1) / kTile : 0;

  // ---- this wave's rows: Q, dO, lse and D = <dO, O>
  const int64_t branch_rows = (int64_t)p.S * p.C * p.Hq;
  const float* outb = gather ? p.o32_g + (int64_t)view * branch_rows * kD : p.o32_f;
  const uint16_t* doutb = gather ? p.dout_g + (int64_t)view * branch_rows * kD : p.dout_f;
  const float* lseb = gather ? p.lse_g + (int64_t)view * branch_rows : p.lse_f;
  DqRows rw;
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    const int n = rb * 32 + 16 * nt + lr;
    const bool valid = has_rows && n < p.R;
    const int j = valid ? n / p.G : 0;
    const int h = g * p.G + (valid ? n % p.G : 0);
    const int64_t orow = ((int64_t)s * p.C + j) * p.Hq + h;
    rw.rowpos[nt] = valid ? L - p.C + j : 0x7FFFFFFF;
    float dsum = 0.f;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int64_t off = orow * kD + 32 * lg + 8 * kk;
      const u32x4 qv = valid ? load16(p.q + off) : u32x4{0u, 0u, 0u, 0u};
      const u32x4 dv = valid ? load16(doutb + off) : u32x4{0u, 0u, 0u, 0u};
      const f32x4 o0 = valid ? *reinterpret_cast<const f32x4*>(outb + off) : f32x4{0.f, 0.f, 0.f, 0.f};
      const f32x4 o1 = valid ? *reinterpret_cast<const f32x4*>(outb + off + 4) : f32x4{0.f, 0.f, 0.f, 0.f};
      rw.qop[nt][kk] = as_bf16x8(qv);
      rw.dop[nt][kk] = as_bf16x8(dv);
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        dsum += bf16_lo(dv[e]) * o0[2 * e] + bf16_hi(dv[e]) * o0[2 * e + 1];
        dsum += bf16_lo(dv[e + 2]) * o1[2 * e] + bf16_hi(dv[e + 2]) * o1[2 * e + 1];
      }
    }
    rw.Dr[nt] = sum_xor32(sum_xor16(dsum));
    const float l2 = valid ? lseb[orow] * kLog2e : INFINITY;
    rw.lse2[nt] = l2 == -INFINITY ? INFINITY : l2;   // a row that saw no key has all-zero weights
  }

  const bool arith = !PAGED && !gather;
  if (!arith) {
    const int nslots = (ntiles + kQRing) * kTile;
    fill_slot_table<PAGED, kQThreads, kQSlotCap>(p.kv, s, g, L, idx_row, e_begin, e_end, nslots, sm.roff, sm.tpos,
                                                 tid);
    __syncthreads();
  }
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
  const uint32_t base16 = arith ? (uint32_t)(((int64_t)s * p.kv.stride_seq + (int64_t)g * p.kv.stride_head) >> 3) : 0u;
  const uint32_t tok16 = (uint32_t)(p.kv.stride_tok >> 3);
  const uint32_t roff_lds = lds_addr(sm.roff), tpos_lds = lds_addr(sm.tpos);
  const uint32_t ring_lds = lds_addr(sm.ring[0]);
  auto arith_rows = [&](int tile, uint32_t (&r)[3]) {
    if (tile >= ntiles) { r[0] = r[1] = r[2] = 0u; return; }   // padding: row 0, a cache-resident address
    const uint32_t r0 = base16 + (uint32_t)(e_begin + kTile * tile) * tok16;
    r[0] = r0 + (uint32_t)rit0 * tok16;
    r[1] = r0 + (uint32_t)rit1 * tok16;
    r[2] = r0 + (uint32_t)rit2 * tok16;
  };
  auto issue = [&](int tile, const uint32_t (&r)[3]) {
    uint8_t* dst = sm.ring[tile % kQRing];
    dq_dma_load(p.kv, r[0], p.max_roff, q0, dst, lane);
    dq_dma_load(p.kv, r[1], p.max_roff, q0 + 1, dst, lane);
    dq_dma_load(p.kv, r[2], p.max_roff, q0 + 2, dst, lane);
  };

  auto stream = [&](auto arith_tag) {
    constexpr bool ARITH = decltype(arith_tag)::value;
    for (int t = 0; t < kQRing - 1; ++t) {
      uint32_t r[3];
      if constexpr (ARITH) {
        arith_rows(t, r);
      } else {
        asm volatile(
            "ds_read_b32 %0, %3\n"
            "ds_read_b32 %1, %4\n"
            "ds_read_b32 %2, %5\n"
            "s_waitcnt lgkmcnt(0)"
            : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2])
            : "v"(roff_lds + 4 * (kTile * t + rit0)), "v"(roff_lds + 4 * (kTile * t + rit1)),
              "v"(roff_lds + 4 * (kTile * t + rit2)));
      }
      issue(t, r);
    }
    int fd_arith = 0;
    if constexpr (ARITH) {
      const int c1 = minpos - e_begin - (kTile - 1);
      const int fd1 = c1 < 0 ? 0 : c1 / kTile + 1;
      const int fd2 = (e_end - e_begin) / kTile;
      fd_arith = fd1 < fd2 ? fd1 : fd2;
    }
    for (int t = 0; t < ntiles; ++t) {
      // this wave's loads of tile t are older than the kQRing-2 tiles issued after it
      asm volatile("s_waitcnt vmcnt(9)\n\ts_barrier" ::: "memory");
      static_assert(3 * (kQRing - 2) == 9, "wait count follows the ring depth");
      const int nxt = t + kQRing - 1;
      const uint32_t src = ring_lds + (uint32_t)(t % kQRing) * kQTileBytes;
      u32x4 kreg[8];
      uint32_t r[3];
      bool dirty;
      u32x4 tp[2];
      if constexpr (ARITH) {
        read8(kreg, src + 16 * lane);
        arith_rows(nxt, r);
        dirty = t >= fd_arith;
      } else {
        const int next0 = kTile * nxt;
        read8_pos_rows(kreg, tp, r, src + 16 * lane, tpos_lds + 4 * (kTile * t + 4 * lg),
                       roff_lds + 4 * (next0 + rit0), roff_lds + 4 * (next0 + rit1), roff_lds + 4 * (next0 + rit2));
        bool bad = false;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int tq = (int)tp[i >> 2][i & 3];
          bad |= tq < 0 || tq > minpos;
        }
        dirty = __builtin_amdgcn_ballot_w64(bad) != 0;
      }
      issue(nxt, r);
      if (has_rows) {
        if constexpr (ARITH) {
          const int slot0 = kTile * t;
          dq_tile_step(acc, rw, kreg, src, lane, p.scale_log2, dirty, [&](int i) {
            const int e = e_begin + slot0 + 16 * (i >> 2) + 4 * lg + (i & 3);
            return e < e_end ? e : -1;
          });
        } else {
          dq_tile_step(acc, rw, kreg, src, lane, p.scale_log2, dirty, [&](int i) { return (int)tp[i >> 2][i & 3]; });
        }
      }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // padding loads land before the block ends
  };
  if (ntiles > 0) {
    if (arith) stream(BoolTag<true>{});
    else stream(BoolTag<false>{});
  }

  // ---- dQ rows 16*nt + lane%16; register i of d-tile dt holds d = 32*(lane/16) + 8*i + dt
  auto write_rows = [&](const f32x4 (&o)[2][8]) {
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const int n = rb * 32 + 16 * nt + lr;
      if (n >= p.R) continue;
      const int j = n / p.G, h = g * p.G + n % p.G;
      float* drow = p.dq + (((int64_t)s * p.C + j) * p.Hq + h) * kD + 32 * lg;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        *reinterpret_cast<f32x4*>(drow + 8 * i) =
            f32x4{o[nt][0][i], o[nt][1][i], o[nt][2][i], o[nt][3][i]} * p.scale;
        *reinterpret_cast<f32x4*>(drow + 8 * i + 4) =
            f32x4{o[nt][4][i], o[nt][5][i], o[nt][6][i], o[nt][7][i]} * p.scale;
      }
    }
  };
  if (p.nb == 1) {
    if (has_rows) write_rows(acc);
    return;
  }

  // ---- publish this wave's partial as record k_rec of its row block: chunk (nt, dt) x lane float4s
  const __amdgpu_buffer_rsrc_t urec =
      make_rsrc(p.part_q + ((int64_t)unit * kQWaves + wave) * p.nb * kRecFloats, (uint32_t)(p.nb * kRecFloats * 4));
  if (has_rows) {
    const uint32_t rec = (uint32_t)k_rec * kRecFloats * 4;
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) store16_coherent(urec, rec + 16 * ((nt * 8 + dt) * kWave + lane), acc[nt][dt]);
  }
  wait_vmem();
  __syncthreads();
  if (tid == 0) sm.last = arrive(counter_line(p.counters, unit), (uint32_t)p.nb);
  __syncthreads();
  if (!sm.last) return;
  if (tid == 0) reset_counter(counter_line(p.counters, unit));
  if (!has_rows) return;
  // sum the row block's partials in (branch, split) order
#pragma unroll
  for (int nt = 0; nt < 2; ++nt)
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) acc[nt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int k = 0; k < p.nb; ++k) {
    const uint32_t rec = (uint32_t)k * kRecFloats * 4;
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) acc[nt][dt] += load16_coherent(urec, rec + 16 * ((nt * 8 + dt) * kWave + lane));
  }
  write_rows(acc);
}

// ---- dK/dV kernel ---------------------------------------------------------------
constexpr int kKWaves = 4;
constexpr int kKThreads = kKWaves * kWave;
constexpr int kPitch = 2 * kD + 16;   // bytes per staged row: the 16-byte pad spreads rows over the banks

struct DkvSmem {
  alignas(16) uint8_t q[32 * kPitch];
  alignas(16) uint8_t dout[32 * kPitch];
  float lse2[32];
  float D[32];
  int32_t cnt[kMaxBwdBlock];   // occurrences of block key c in the branch's key list
  int32_t last;
};

__device__ inline u32x4 lds_read16(const uint8_t* base, uint32_t off) {
  return *reinterpret_cast<const u32x4*>(base + off);
}

template <bool PAGED>
__global__ __launch_bounds__(kKThreads) void dkv_kernel(AttnBwdParams p) {
  __shared__ DkvSmem sm;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lg = lane >> 4, lr = lane & 15;
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int br = bid % p.nbr;
  const int pair = bid / p.nbr;            // s * Hkv + g
  const int g = pair % p.Hkv, s = pair / p.Hkv;
  const bool gather = br < p.V;
  const int L = seq_len(p.kv, s);
  const int C = p.C, t0 = L - C;           // block row c sits at position t0 + c

  // ---- key multiplicities of the branch
  for (int c = tid; c < C; c += kKThreads) sm.cnt[c] = (!gather && t0 + c >= 0) ? 1 : 0;
  __syncthreads();
  if (gather) {
    const int32_t* idx_row = p.idx + (((int64_t)br * p.S + s) * p.Hkv + g) * p.ld_idx;
    int n = p.nsel[br * p.S + s];
    n = n < 0 ? 0 : (n > p.ld_idx ? p.ld_idx : n);
    for (int e = tid; e < n; e += kKThreads) {
      const int t = idx_row[e];
      if (t >= 0 && t < L && t >= t0) atomicAdd(&sm.cnt[t - t0], 1);
    }
    __syncthreads();
  }

  const int64_t branch_rows = (int64_t)p.S * C * p.Hq;
  const float* outb = gather ? p.o32_g + (int64_t)br * branch_rows * kD : p.o32_f;
  const uint16_t* doutb = gather ? p.dout_g + (int64_t)br * branch_rows * kD : p.dout_f;
  const float* lseb = gather ? p.lse_g + (int64_t)br * branch_rows : p.lse_f;
  const int nkt = (C + 15) / 16;
  const int nrt = (p.R + 31) / 32;
  float* rec_k = p.part_kv + ((int64_t)pair * p.nbr + br) * C * 2 * kD;
  float* rec_v = rec_k + (int64_t)C * kD;
  const bool direct = p.nbr == 1;
  const __amdgpu_buffer_rsrc_t rrec = make_rsrc(rec_k, (uint32_t)(C * 2 * kD * 4));
  float* out_k = direct ? p.dk + (int64_t)s * C * p.Hkv * kD : rec_k;
  float* out_v = direct ? p.dv + (int64_t)s * C * p.Hkv * kD : rec_v;
  const int64_t out_stride = direct ? (int64_t)p.Hkv * kD : kD;   // floats between block rows
  const int64_t out_head = direct ? (int64_t)g * kD : 0;

  for (int kt0 = 0; kt0 < nkt; kt0 += kKWaves) {
    const int kt = kt0 + wave;
    const int c = kt * 16 + lr;                        // this lane's block key
    const bool kvalid = kt < nkt && c < C && t0 + c >= 0;
    const int mult = kvalid ? sm.cnt[c] : 0;
    const bool active = __builtin_amdgcn_ballot_w64(mult > 0) != 0;
    // B operands: K_blk^T and V_blk^T, lane l feeding key l%16 with d slots 32*(l/16) + 8*j ..
    bf16x8 kop[4], vop[4];
    {
      int64_t o = -1;
      if (kvalid && mult > 0) o = row_offset<PAGED>(p.kv, s, g, t0 + c);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        kop[j] = as_bf16x8(o >= 0 ? load16(p.kv.k + o + 32 * lg + 8 * j) : u32x4{0u, 0u, 0u, 0u});
        vop[j] = as_bf16x8(o >= 0 ? load16(p.kv.v + o + 32 * lg + 8 * j) : u32x4{0u, 0u, 0u, 0u});
      }
    }
    f32x4 dk[8], dv[8];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) dk[dt] = dv[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int rt = 0; rt < nrt; ++rt) {
      __syncthreads();   // the previous row tile's reads are done
      // stage Q and dO of rows 32*rt .. +31 (row-major, padded) with lse and D
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int ci = tid + kKThreads * u;
        const int r = ci >> 4, cc = ci & 15;
        const int n = 32 * rt + r;
        const bool valid = n < p.R;
        const int j = valid ? n / p.G : 0, h = g * p.G + (valid ? n % p.G : 0);
        const int64_t orow = ((int64_t)s * C + j) * p.Hq + h;
        const int64_t off = orow * kD + 8 * cc;
        const u32x4 qv = valid ? load16(p.q + off) : u32x4{0u, 0u, 0u, 0u};
        const u32x4 dv4 = valid ? load16(doutb + off) : u32x4{0u, 0u, 0u, 0u};
        const f32x4 o0 = valid ? *reinterpret_cast<const f32x4*>(outb + off) : f32x4{0.f, 0.f, 0.f, 0.f};
        const f32x4 o1 = valid ? *reinterpret_cast<const f32x4*>(outb + off + 4) : f32x4{0.f, 0.f, 0.f, 0.f};
        *reinterpret_cast<u32x4*>(sm.q + r * kPitch + 16 * cc) = qv;
        *reinterpret_cast<u32x4*>(sm.dout + r * kPitch + 16 * cc) = dv4;
        float dsum = 0.f;
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          dsum += bf16_lo(dv4[e]) * o0[2 * e] + bf16_hi(dv4[e]) * o0[2 * e + 1];
          dsum += bf16_lo(dv4[e + 2]) * o1[2 * e] + bf16_hi(dv4[e + 2]) * o1[2 * e + 1];
        }
        dsum = sum16(dsum);
        if (cc == 0) {
          sm.D[r] = dsum;
          const float l2 = valid ? lseb[orow] * kLog2e : INFINITY;
          sm.lse2[r] = l2 == -INFINITY ? INFINITY : l2;
        }
      }
      __syncthreads();
      if (!active) continue;

      // S and dP with rows on the M side: lane l holds rows 16*sub + 4*(l/16) + i of key l%16
      f32x4 sp[2], dp[2];
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
        f32x4 a = {0.f, 0.f, 0.f, 0.f}, b = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint32_t off = (16 * sub + lr) * kPitch + 64 * lg + 16 * j;
          a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(lds_read16(sm.q, off)), kop[j], a, 0, 0, 0);
          b = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(lds_read16(sm.dout, off)), vop[j], b, 0, 0, 0);
        }
        sp[sub] = a;
        dp[sub] = b;
      }
      u32x4 pw, dsw, pwl, dswl;
#pragma unroll
      for (int i2 = 0; i2 < 4; ++i2) {
        float pv[2], dsv[2];
#pragma unroll
        for (int e2 = 0; e2 < 2; ++e2) {
          const int slot = 2 * i2 + e2;                       // k-slot: row 16*(slot/4) + 4*lg + slot%4
          const int sub = slot >> 2, i = slot & 3;
          const int r = 16 * sub + 4 * lg + i;
          const int n = 32 * rt + r;
          const bool vis = mult > 0 && n < p.R && c <= n / p.G;
          const float pr = vis ? __builtin_amdgcn_exp2f(fmaf(sp[sub][i], p.scale_log2, -sm.lse2[r])) : 0.f;
          pv[e2] = pr;
          dsv[e2] = pr * (dp[sub][i] - sm.D[r]);
        }
        pw[i2] = pack_bf16x2(pv[0], pv[1]);
        dsw[i2] = pack_bf16x2(dsv[0], dsv[1]);
        pwl[i2] = pack_bf16x2(pv[0] - bf16_lo(pw[i2]), pv[1] - bf16_hi(pw[i2]));
        dswl[i2] = pack_bf16x2(dsv[0] - bf16_lo(dsw[i2]), dsv[1] - bf16_hi(dsw[i2]));
      }
      // transposed operands: rows 16*h + 4*lg + i (register 4*h + i), 16 bytes at d = 8*lr
      u32x4 qt[8], dot[8];
#pragma unroll
      for (int x = 0; x < 8; ++x) {
        const uint32_t off = (16 * (x >> 2) + 4 * lg + (x & 3)) * kPitch + 16 * lr;
        qt[x] = lds_read16(sm.q, off);
        dot[x] = lds_read16(sm.dout, off);
      }
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        const bf16x8 a_do = vt_operand(dot, dt), a_q = vt_operand(qt, dt);
        dv[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_do, as_bf16x8(pw), dv[dt], 0, 0, 0);
        dv[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_do, as_bf16x8(pwl), dv[dt], 0, 0, 0);
        dk[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_q, as_bf16x8(dsw), dk[dt], 0, 0, 0);
        dk[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_q, as_bf16x8(dswl), dk[dt], 0, 0, 0);
      }
    }

    // block key c: register i of d-tile dt holds d = 32*lg + 8*i + dt; a key listed m times counts m times
    if (kt < nkt && c < C) {
      const float mk = (float)mult * (direct ? p.scale : 1.f), mv = (float)mult;
      float* kr = out_k + (int64_t)c * out_stride + out_head + 32 * lg;
      float* vr = out_v + (int64_t)c * out_stride + out_head + 32 * lg;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const f32x4 k0 = f32x4{dk[0][i], dk[1][i], dk[2][i], dk[3][i]} * mk;
        const f32x4 k1 = f32x4{dk[4][i], dk[5][i], dk[6][i], dk[7][i]} * mk;
        const f32x4 v0 = f32x4{dv[0][i], dv[1][i], dv[2][i], dv[3][i]} * mv;
        const f32x4 v1 = f32x4{dv[4][i], dv[5][i], dv[6][i], dv[7][i]} * mv;
        if (direct) {
          *reinterpret_cast<f32x4*>(kr + 8 * i) = k0;
          *reinterpret_cast<f32x4*>(kr + 8 * i + 4) = k1;
          *reinterpret_cast<f32x4*>(vr + 8 * i) = v0;
          *reinterpret_cast<f32x4*>(vr + 8 * i + 4) = v1;
        } else {
          const uint32_t ok = (uint32_t)((c * kD + 32 * lg + 8 * i) * 4), ov = ok + (uint32_t)(C * kD * 4);
          store16_coherent(rrec, ok, k0);
          store16_coherent(rrec, ok + 16, k1);
          store16_coherent(rrec, ov, v0);
          store16_coherent(rrec, ov + 16, v1);
        }
      }
    }
  }
  if (direct) return;

  // ---- the last branch of (s, g) to finish adds the branches' partials in branch order
  wait_vmem();
  __syncthreads();
  uint32_t* ctr = counter_line(p.counters, (int64_t)p.units + pair);
  if (tid == 0) sm.last = arrive(ctr, (uint32_t)p.nbr);
  __syncthreads();
  if (!sm.last) return;
  if (tid == 0) reset_counter(ctr);
  const float* recs = p.part_kv + (int64_t)pair * p.nbr * C * 2 * kD;
  const __amdgpu_buffer_rsrc_t rr = make_rsrc(recs, (uint32_t)((int64_t)p.nbr * C * 2 * kD * 4));
  const int chunks = C * 2 * kD / 4;                 // float4s of one branch record
  for (int q = tid; q < chunks; q += kKThreads) {
    f32x4 sum = {0.f, 0.f, 0.f, 0.f};
    for (int b = 0; b < p.nbr; ++b) sum += load16_coherent(rr, (uint32_t)(((int64_t)b * chunks + q) * 16));
    const int fl = 4 * q;                            // float index within [dk | dv] of one branch
    const bool isv = fl >= C * kD;
    const int rem = isv ? fl - C * kD : fl;
    const int cc = rem / kD, d = rem % kD;
    float* dst = (isv ? p.dv : p.dk) + (((int64_t)s * C + cc) * p.Hkv + g) * kD + d;
    *reinterpret_cast<f32x4*>(dst) = isv ? sum : sum * p.scale;
  }
}

}  // namespace

AttnBwdPlan plan_attn_bwd(int S, int Hkv, int Hq, int C, int num_views, int ld_idx, int max_L, bool with_full,
                          bool paged, bool with_dkv) {
  AttnBwdPlan pl{};
  const int G = Hq / Hkv;
  pl.R = C * G;
  pl.n_rb = (pl.R + 31) / 32;
  pl.n_rg = (pl.n_rb + kQWaves - 1) / kQWaves;
  pl.units = S * Hkv * pl.n_rg;
  const int64_t units_g = (int64_t)num_views * pl.units, units_f = with_full ? pl.units : 0;
  auto round_up = [](int64_t x, int64_t m) { return (x + m - 1) / m * m; };
  const int64_t work = units_g * ld_idx + units_f * max_L;
  const int64_t g_all = round_up(ld_idx > 0 ? ld_idx : 1, kTile), f_all = round_up(max_L > 0 ? max_L : 1, kTile);
  // keys per split: from work / kTargetBlocks up, the smallest multiple of the tile that keeps the
  // launch to one workgroup per CU; view splits and paged full splits are bound by the slot table
  int64_t kps = round_up((work + kTargetBlocks - 1) / kTargetBlocks, kTile);
  if (kps < kTile) kps = kTile;
  int64_t kg, kf, blocks;
  for (;;) {
    kg = kps < g_all ? kps : g_all;
    if (kg > kMaxSplitKeys) kg = kMaxSplitKeys;
    kf = kps < f_all ? kps : f_all;
    if (paged && kf > kMaxSplitKeys) kf = kMaxSplitKeys;
    blocks = units_g * ((g_all + kg - 1) / kg) + units_f * ((f_all + kf - 1) / kf);
    if (blocks <= kTargetBlocks || (kps >= g_all && kps >= f_all)) break;
    kps += kTile;
  }
  pl.kps_g = (int)kg;
  pl.kps_f = (int)kf;
  pl.nsplit_g = ld_idx > 0 ? (int)((ld_idx + kg - 1) / kg) : 1;
  pl.nsplit_f = max_L > 0 ? (int)((max_L + kf - 1) / kf) : 1;
  pl.nb = num_views * pl.nsplit_g + (with_full ? pl.nsplit_f : 0);
  pl.nblk_g = (int)(units_g * pl.nsplit_g);
  pl.nblk_q = (int)(units_g * pl.nsplit_g + units_f * pl.nsplit_f);
  pl.nbr = num_views + (with_full ? 1 : 0);
  pl.counter_bytes = BD_WS_COUNTER_BYTES;
  pl.q_record_bytes = pl.nb > 1 ? align256(sizeof(float) * kRecFloats * (size_t)pl.units * kQWaves * pl.nb) : 0;
  pl.kv_record_bytes =
      with_dkv && pl.nbr > 1 ? align256(sizeof(float) * (size_t)S * Hkv * pl.nbr * C * 2 * kD) : 0;
  pl.ws_bytes = pl.counter_bytes + pl.q_record_bytes + pl.kv_record_bytes;
  return pl;
}

hipError_t launch_attn_bwd(const AttnBwdParams& p, const AttnBwdPlan& pl, bool paged, hipStream_t stream) {
  if (pl.nblk_q > 0) {
    if (paged) hipLaunchKernelGGL(dq_kernel<true>, dim3(pl.nblk_q), dim3(kQThreads), 0, stream, p);
    else hipLaunchKernelGGL(dq_kernel<false>, dim3(pl.nblk_q), dim3(kQThreads), 0, stream, p);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (p.dk) {
    const int nblk = p.S * p.Hkv * p.nbr;
    if (paged) hipLaunchKernelGGL(dkv_kernel<true>, dim3(nblk), dim3(kKThreads), 0, stream, p);
    else hipLaunchKernelGGL(dkv_kernel<false>, dim3(nblk), dim3(kKThreads), 0, stream, p);
    return hipGetLastError();
  }
  return hipSuccess;
}

}  // namespace bd
