// Budgeted KV selection (Alg. 2 "sparsify"; Sec. 3.4: keep the entries with
// the largest cumulative attention weight).
//
// Three launches:
//   1. score pass 1 (skipped when the caller gives the window rows'
//      log-sum-exp): every (sequence, KV head, row block, key split) computes
//      the running max and sum of exp of each observation row over its keys;
//   2. score pass 2: merges those statistics into each row's log-sum-exp and
//      streams K again, adding every row's normalised weight of every key
//      into that key's column sum (complete within a row block, so no atomics);
//   3. top-B: one 1024-thread workgroup per (sequence, KV head) sums the row
//      blocks, max-pools the prefix (or sums its chunks), finds the K-th
//      largest candidate score with a radix select over the float bit patterns
//      (digits of 8, 11 and 12 bits; scores are non-negative, so the bits order
//      like the values), and compacts the chosen positions in ascending order;
//      ties at the threshold take the lowest positions, then the window is
//      appended.
//
// The scoring product is a real dense contraction ((W*G) x 128 x L per
// (s, g)), so it runs on MFMA with the attention kernel's orientation: keys on
// the M side, observation rows on the N side.  Lane l then holds 4 keys of
// row l%16: row statistics stay lane-local, and a key's column sum is a
// 16-lane DPP reduction.

#include <type_traits>

#include "bd_common.hpp"
#include "bd_kernels.hpp"

namespace bd {
namespace {

constexpr int kWaves = 8;                        // two per SIMD: one wave's MFMA and loads overlap another's VALU
constexpr int kThreads = kWaves * kWave;
constexpr int kTile = 32;                        // keys per wave iteration (two MFMA sub-tiles of 16)
constexpr int kTileLoads = 8;                    // 16-byte loads per lane per tile
constexpr int kTileBytes = kTileLoads * kWave * 16;
constexpr int kRing = 2;                         // tile slots per wave: one in flight while one is computed
constexpr int kMaxPagedKeys = 4096;              // keys per workgroup through the paged slot table
constexpr int kSlotCap = kMaxPagedKeys + kRing * kWaves * kTile;
constexpr int kStatRows = 128;                   // stats record stride (rows)
constexpr int kTargetBlocks = 256;               // one workgroup per CU
constexpr int kTopkThreads = 1024;
constexpr int kMaxPerThread = BD_SELECT_MAX_PREFIX / kTopkThreads;   // 32
constexpr int kHistWords = 4096;                // radix histogram words: bins x copies of each digit
// Radix digits of the top-B keys, most significant first (bits, lowest bit, histogram copies).
constexpr int kDigits = 3;
__device__ inline int digit_bits(int i) { return i == 0 ? 8 : (i == 1 ? 11 : 12); }
__device__ inline int digit_shift(int i) { return i == 0 ? 23 : (i == 1 ? 12 : 0); }
__device__ inline int digit_copies(int i) { return i == 0 ? 16 : (i == 1 ? 2 : 1); }
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kSlack = 8.f;                    // lazy-rescale headroom of the pass-1 sums, log2 units

__device__ inline void merge_ml(float& m, float& l, float m2, float l2) {
  const float M = fmaxf(m, m2);
  if (M == -INFINITY) { m = M; l = 0.f; return; }
  l = l * exp2f(m - M) + l2 * exp2f(m2 - M);
  m = M;
}

// Every kernel argument requested at entry: fetched where first used they took four or five round
// trips in a row before the first data load.  The statements touch no memory and return 0, which
// the caller adds to its block index.
__device__ inline int fetch_select_args(const SelectParams& p) {
  int z0, z1, z2;
  asm("s_mov_b32 %0, 0" : "=s"(z0) : "s"(p.kv.k), "s"(p.kv.seq_lens), "s"(p.kv.page_table), "s"(p.kv.stride_seq),
      "s"(p.kv.stride_head), "s"(p.kv.stride_tok), "s"(p.kv.stride_page), "s"(p.kv.max_seq_len), "s"(p.kv.page_size),
      "s"(p.kv.max_pages_per_seq), "s"(p.kv.num_pages));
  asm("s_mov_b32 %0, 0" : "=s"(z1) : "s"(z0), "s"(p.q_win), "s"(p.lse_win), "s"(p.S), "s"(p.Hkv), "s"(p.Hq), "s"(p.G),
      "s"(p.W), "s"(p.budget), "s"(p.pool_kernel), "s"(p.chunk), "s"(p.keep), "s"(p.ld), "s"(p.R), "s"(p.n_rb));
  asm("s_mov_b32 %0, 0" : "=s"(z2) : "s"(z1), "s"(p.nsplit), "s"(p.kps), "s"(p.max_L), "s"(p.scale_log2),
      "s"(p.max_roff), "s"(p.stats), "s"(p.raw_part), "s"(p.raw), "s"(p.idx_out), "s"(p.nsel_out), "s"(p.page_arith));
  return z2;
}

template <int NT, bool PAGED>
struct ScoreSmem {
  alignas(16) uint8_t ring[kWaves][kRing][kTileBytes];   // per-wave K tile slots filled by DMA
  alignas(16) int32_t roff[PAGED ? kSlotCap : 4];        // paged: row offset (16-byte units) per key slot
  float m[kWaves][16 * NT];
  float l[kWaves][16 * NT];
  float lse2[16 * NT];
};

__device__ inline void dma16(const uint16_t* g, uint8_t* l) {
  __builtin_amdgcn_global_load_lds((const void*)g, (__attribute__((address_space(3))) void*)l, 16, 0, 0);
}

// Direct-to-LDS loads of one K tile: load q (sub-tile q/4, k-step q%4) of a lane lands at
// dst + q*1 KiB + 16*lane; the lane's rows are r[sub] (16-byte units, clamped to the layout).
__device__ inline void dma_ktile(const uint16_t* k, const uint32_t (&r)[2], uint32_t max_roff, uint8_t* dst, int lane) {
  const int lg = lane >> 4;
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) {
    const uint32_t ro = r[sub] < max_roff ? r[sub] : max_roff;
    const uint16_t* kr = k + ((uint64_t)ro << 3) + 32 * lg;
#pragma unroll
    for (int j = 0; j < 4; ++j) dma16(kr + 8 * j, dst + (4 * sub + j) * 1024);
  }
}

// Copy a landed K tile into registers (loads and their wait in one asm statement: the compiler
// would otherwise wait for every direct-to-LDS load in flight before any LDS read).
__device__ inline void read_ktile(u32x4 (&t)[2][4], uint32_t src, int lane) {
  const uint32_t a = src + 16 * lane;
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
      : "=&v"(t[0][0]), "=&v"(t[0][1]), "=&v"(t[0][2]), "=&v"(t[0][3]), "=&v"(t[1][0]), "=&v"(t[1][1]),
        "=&v"(t[1][2]), "=&v"(t[1][3])
      : "v"(a));
}

// Row offsets of a paged tile's two lane rows from the slot table.
__device__ inline void read_krows(uint32_t (&r)[2], uint32_t roff_lds, int slot0, int lane) {
  const uint32_t a = roff_lds + 4 * (slot0 + (lane & 15));
  asm volatile(
      "ds_read_b32 %0, %2\n"
      "ds_read_b32 %1, %2 offset:64\n"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(r[0]), "=&v"(r[1])
      : "v"(a));
}

// One pass over the causal key range of (sequence, KV head, row block, split).  Each wave streams
// every kWaves-th 32-key tile through a kRing-deep ring of LDS slots.
//   PASS 1: per observation row, running max and sum of exp of the scaled logits;
//   PASS 2: every key's column sum of the rows' normalised weights (complete within the row
//           block: one plain store per key).
template <int NT, bool PAGED, int PASS>
__global__ __launch_bounds__(kThreads) void score_kernel(SelectParams p) {
  __shared__ ScoreSmem<NT, PAGED> sm;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lg = lane >> 4, lr = lane & 15;
  const int bid = xcd_remap(blockIdx.x + fetch_select_args(p), gridDim.x);
  const int rb = bid % p.n_rb;
  const int rest = bid / p.n_rb;
  const int split = rest % p.nsplit;
  const int pair = rest / p.nsplit;
  const int g = pair % p.Hkv, s = pair / p.Hkv;
  const int L = seq_len(p.kv, s);
  if (p.budget >= L) return;               // whole cache kept: nothing to score
  const int k0 = split * p.kps;
  int k1 = k0 + p.kps;
  if (k1 > L) k1 = L;
  const int64_t stat_base = (((int64_t)pair * p.n_rb + rb) * p.nsplit) * kStatRows * 2;

  // observation rows of this lane: n = rb*16*NT + 16*nt + lane%16 -> (window row i, head h)
  bf16x8 qop[NT][4];
  int rowpos[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int n = rb * 16 * NT + 16 * nt + lr;
    const bool valid = n < p.R;
    const int i = valid ? n / p.G : 0;
    const int h = g * p.G + (valid ? n % p.G : 0);
    rowpos[nt] = valid ? L - p.W + i : -1;          // padded rows see no key
    const uint16_t* qrow = p.q_win + (((int64_t)s * p.W + i) * p.Hq + h) * kD + 32 * lg;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) qop[nt][kk] = as_bf16x8(valid ? load16(qrow + 8 * kk) : u32x4{0u, 0u, 0u, 0u});
  }

  const int ntiles = k1 > k0 ? (k1 - k0 + kTile - 1) / kTile : 0;
  // pages holding whole 16-key sub-tiles (page_size a multiple of 16, host-checked): a table of page
  // offsets, one entry per page; k / page_size is computed as (k / 16) / (page_size / 16), exact for
  // keys below 2^26 (host-checked); k0 is a multiple of kWaves * kTile
  const bool page_arith = PAGED && p.page_arith != 0;
  const int psub = PAGED ? p.kv.page_size >> 4 : 1;
  const float inv_psub = __builtin_amdgcn_rcpf((float)psub);
  const int page0 = page_arith ? div_small(k0 >> 4, psub, inv_psub) : 0;
  if (page_arith) {
    // entry j: offset (16-byte units) of page page0 + j for head g, 0 for a page outside the pool (its
    // keys read pool rows and score as whatever those hold); all page-table loads issued first
    constexpr int kPer = (kSlotCap + kThreads - 1) / kThreads;
    const int npg = k1 > k0 ? div_small((k1 - 1) >> 4, psub, inv_psub) - page0 + 1 : 0;
    const int32_t* prow = p.kv.page_table + (int64_t)s * p.kv.max_pages_per_seq + page0;
    int pg[kPer];
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int j = tid + k * kThreads;
      pg[k] = j < npg ? prow[j] : -1;
    }
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int j = tid + k * kThreads;
      if (j < npg)
        sm.roff[j] = (unsigned)pg[k] < (unsigned)p.kv.num_pages
                         ? (int)(((int64_t)pg[k] * p.kv.stride_page + (int64_t)g * p.kv.stride_head) >> 3)
                         : 0;
    }
  } else if constexpr (PAGED) {
    // slot table of this split: all page-table loads issued before any result is used; padding
    // slots (past the split) hold row 0, a safe, cache-resident address
    constexpr int kPer = (kSlotCap + kThreads - 1) / kThreads;
    int pg[kPer];
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int t = k0 + tid + k * kThreads;
      pg[k] = t < k1 ? p.kv.page_table[(int64_t)s * p.kv.max_pages_per_seq + t / p.kv.page_size] : -1;
    }
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int i = tid + k * kThreads;
      if (i < kSlotCap) {
        const int t = k0 + i;
        int64_t o = 0;
        if ((unsigned)pg[k] < (unsigned)p.kv.num_pages)
          o = (int64_t)pg[k] * p.kv.stride_page + (int64_t)g * p.kv.stride_head +
              (int64_t)(t % p.kv.page_size) * p.kv.stride_tok;
        sm.roff[i] = (int)(o >> 3);
      }
    }
  }

  // lse of each row (pass 2): the caller's, or merged from the pass-1 statistics.  Padded rows get
  // +inf, so their weights are exactly zero even where no mask is applied.
  // pass 1 per row: reference mu (log2 units, 0 until the first visible key), sum rl of exp2 relative
  // to it, and the raw (unscaled) logit above which mu is raised
  float rm[NT], rl[NT], rthr[NT], lse2[NT];
  if constexpr (PASS == 2) {
    if (tid < 16 * NT) {
      const int n = rb * 16 * NT + tid;
      float v = INFINITY;
      if (n < p.R) {
        if (p.lse_win) {
          const int i = n / p.G, h = g * p.G + n % p.G;
          v = p.lse_win[((int64_t)s * p.W + i) * p.Hq + h] * kLog2e;
        } else {
          float m = -INFINITY, l = 0.f;
          for (int sp = 0; sp < p.nsplit; ++sp) {
            const float* st = p.stats + stat_base + ((int64_t)sp * kStatRows + tid) * 2;
            merge_ml(m, l, st[0], st[1]);
          }
          v = l > 0.f ? m + __log2f(l) : INFINITY;   // empty row contributes nothing
        }
      }
      sm.lse2[tid] = v;
    }
  } else {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) { rm[nt] = 0.f; rl[nt] = 0.f; rthr[nt] = -INFINITY; }
  }
  __syncthreads();
  if constexpr (PASS == 2) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) lse2[nt] = sm.lse2[16 * nt + lr];
  }

  // tiles whose keys all lie inside the split and at or before the block's earliest row position
  // need no mask
  const int minpos = L - p.W + (rb * 16 * NT) / p.G;
  int first_dirty;
  {
    const int c1 = minpos - k0 - (kTile - 1);
    const int fd1 = c1 < 0 ? 0 : c1 / kTile + 1;
    const int fd2 = (k1 - k0) / kTile;
    first_dirty = fd1 < fd2 ? fd1 : fd2;
  }

  float* raw_part = p.raw_part + ((int64_t)pair * p.n_rb + rb) * p.max_L;

  // Scores of one 16-key sub-tile against the 16*NT rows; keys tb .. tb+3 belong to this lane.
  auto sub_products = [&](f32x4 (&acc)[NT], const u32x4 (&kr)[4]) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      f32x4 a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < 4; ++j) a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kr[j]), qop[nt][j], a, 0, 0, 0);
      acc[nt] = a;
    }
  };
  // Causal and split mask of a sub-tile.  Only tiles that can hold a masked key call it: a mask
  // behind a runtime flag was if-converted, and every tile paid it (a compare, a select and a mask
  // merge per score: a third of the loop's VALU instructions).
  auto sub_mask = [&](f32x4 (&acc)[NT], int tb) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = tb + i;
        if (!(t < k1 && t <= rowpos[nt])) acc[nt][i] = -INFINITY;
      }
  };

  // Pass 1 over a 32-key tile: per-lane running sums with a lazily raised reference, so weights stay
  // <= 2^kSlack.  Both sub-tiles' products come first and one check covers the tile: it compares raw
  // logits with a per-row threshold, and the raise is a wave-uniform branch (the common tile pays
  // max and compare instructions, no extra exponential).  One branch per tile instead of one per
  // sub-tile leaves the scheduler one block of 64 products to interleave with the exponentials.
  auto pass1_tile = [&](const u32x4 (&kt)[2][4], int tb, auto dirty_tag) {
    f32x4 acc[2][NT];
    sub_products(acc[0], kt[0]);
    sub_products(acc[1], kt[1]);
    if constexpr (decltype(dirty_tag)::value) {
      sub_mask(acc[0], tb);
      sub_mask(acc[1], tb + 16);
    }
    float mx[NT];
    bool raise = false;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      mx[nt] = fmaxf(fmaxf(fmaxf(acc[0][nt][0], acc[0][nt][1]), fmaxf(acc[0][nt][2], acc[0][nt][3])),
                     fmaxf(fmaxf(acc[1][nt][0], acc[1][nt][1]), fmaxf(acc[1][nt][2], acc[1][nt][3])));
      raise |= mx[nt] > rthr[nt];
    }
    if (__builtin_expect(__builtin_amdgcn_ballot_w64(raise) != 0, 0)) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        if (mx[nt] > rthr[nt]) {
          const float m2 = mx[nt] * p.scale_log2;    // scale > 0: the max commutes with it
          rl[nt] = rl[nt] > 0.f ? rl[nt] * exp2f(rm[nt] - m2) : 0.f;
          rm[nt] = m2;
          rthr[nt] = (m2 + kSlack) / p.scale_log2;
        }
      }
    }
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) rl[nt] += __builtin_amdgcn_exp2f(fmaf(acc[sub][nt][i], p.scale_log2, -rm[nt]));
  };

  // Pass 2 over a 16-key sub-tile: each key's column sum of the rows' normalised weights.  After the
  // 16-lane reduction every lane of a row holds the same four sums (each step adds a lane pair in
  // both orders), so in a mask-free tile all 64 lanes store, four lanes per key with equal bits,
  // and no branch splits the loop body: the next sub-tile's products can overlap this one's sums.
  auto pass2_sub = [&](const u32x4 (&kr)[4], int tb, auto dirty_tag) {
    constexpr bool dirty = decltype(dirty_tag)::value;
    f32x4 acc[NT];
    sub_products(acc, kr);
    if constexpr (dirty) sub_mask(acc, tb);
    float col[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) col[i] = __builtin_amdgcn_exp2f(fmaf(acc[0][i], p.scale_log2, -lse2[0]));
#pragma unroll
    for (int nt = 1; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) col[i] += __builtin_amdgcn_exp2f(fmaf(acc[nt][i], p.scale_log2, -lse2[nt]));
#pragma unroll
    for (int i = 0; i < 4; ++i) col[i] = sum16(col[i]);
    // opaque to the compiler, which would otherwise finish the reduction only for the column a lane
    // stores, behind branches on the lane index
    asm("" : "+v"(col[0]), "+v"(col[1]), "+v"(col[2]), "+v"(col[3]));
    const int q = lr & 3;
    const float v01 = (q & 1) ? col[1] : col[0], v23 = (q & 1) ? col[3] : col[2];
    const float v = (q & 2) ? v23 : v01;
    const int t = tb + q;
    if constexpr (dirty) {
      if (lr < 4 && t < k1) raw_part[t] = v;
    } else {
      raw_part[t] = v;                     // a mask-free tile lies inside the split: t < k1
    }
  };

  if (wave < ntiles) {
    const uint32_t ring_lds = lds_addr(sm.ring[wave][0]);
    const uint32_t roff_lds = lds_addr(sm.roff);
    const uint32_t base16 = PAGED ? 0u : (uint32_t)(((int64_t)s * p.kv.stride_seq + (int64_t)g * p.kv.stride_head) >> 3);
    const uint32_t tok16 = (uint32_t)(p.kv.stride_tok >> 3);
    // pass 2 takes its tiles last first: pass 1 read them first to last, so the most recent (still in
    // the memory-side cache) are read before the lines pass 1 read first are replaced
    auto real = [&](int it) { return PASS == 2 ? ntiles - 1 - it : it; };
    auto issue = [&](int tile, int slot) {
      uint32_t r[2];
      if constexpr (PAGED) {
        if (tile >= ntiles) {
          r[0] = r[1] = 0u;
        } else if (page_arith) {
          // sub-tile h (keys tb+16h .. +15) lies in one page: its offset + (key mod page_size) rows
          const int tb = k0 + kTile * real(tile);
          uint32_t a[2], w[2], b[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int t = tb + 16 * h;
            const int pi = div_small(t >> 4, psub, inv_psub);
            a[h] = roff_lds + 4 * (uint32_t)(t < k1 ? pi - page0 : 0);   // past the split: entry 0, masked
            w[h] = (uint32_t)(t - pi * p.kv.page_size);
          }
          asm volatile(
              "ds_read_b32 %0, %2\n"
              "ds_read_b32 %1, %3\n"
              "s_waitcnt lgkmcnt(0)"
              : "=&v"(b[0]), "=&v"(b[1])
              : "v"(a[0]), "v"(a[1]));
#pragma unroll
          for (int h = 0; h < 2; ++h) r[h] = b[h] + (w[h] + (uint32_t)lr) * tok16;
        } else {
          read_krows(r, roff_lds, kTile * real(tile), lane);
        }
      } else if (tile >= ntiles) {
        r[0] = r[1] = 0u;                  // padding: row 0, a safe, cache-resident address
      } else {
        const uint32_t r0 = base16 + (uint32_t)(k0 + kTile * real(tile)) * tok16;
        r[0] = r0 + (uint32_t)lr * tok16;
        r[1] = r0 + (uint32_t)(16 + lr) * tok16;
      }
      dma_ktile(p.kv.k, r, p.max_roff, sm.ring[wave][slot], lane);
    };
#pragma unroll
    for (int q = 0; q < kRing; ++q) issue(wave + kWaves * q, q);
    u32x4 kt[2][4];
    int j = 0;
    // step j of this wave (tile wave + kWaves*j); true after its last tile
    auto step = [&](auto dirty_tag) -> bool {
      const int it = wave + kWaves * j, slot = j % kRing;
      // the tile about to be read was issued (kRing-1) tiles before the newest
      static_assert(kRing == 2, "the wait below assumes one tile (8 loads) issued after the one read");
      asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
      read_ktile(kt, ring_lds + slot * kTileBytes, lane);
      issue(it + kRing * kWaves, slot);
      const int tb = k0 + kTile * real(it) + 4 * lg;
      if constexpr (PASS == 1) {
        pass1_tile(kt, tb, dirty_tag);
      } else {
        pass2_sub(kt[0], tb, dirty_tag);
        pass2_sub(kt[1], tb + 16, dirty_tag);
      }
      ++j;
      return it + kWaves >= ntiles;
    };
    // a wave's tiles increase in pass 1, so its mask-free ones come first; in pass 2 they come last
    bool last = false;
    if constexpr (PASS == 1) {
      while (!last && wave + kWaves * j < first_dirty) last = step(std::integral_constant<bool, false>{});
      while (!last) last = step(std::integral_constant<bool, true>{});
    } else {
      while (!last && real(wave + kWaves * j) >= first_dirty) last = step(std::integral_constant<bool, true>{});
      while (!last) last = step(std::integral_constant<bool, false>{});
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // padding loads land before the block ends
  }

  if constexpr (PASS == 1) {
    // merge the 4 lane groups, then the waves, and publish per-row (max, sum) of this split
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      if (!(rl[nt] > 0.f)) rm[nt] = -INFINITY;   // no visible key: the empty (max, sum)
#pragma unroll
      for (int m = 16; m <= 32; m <<= 1) {
        const float m2 = shfl_xor_f(rm[nt], m), l2 = shfl_xor_f(rl[nt], m);
        merge_ml(rm[nt], rl[nt], m2, l2);
      }
      if (lg == 0) {
        sm.m[wave][16 * nt + lr] = rm[nt];
        sm.l[wave][16 * nt + lr] = rl[nt];
      }
    }
    __syncthreads();
    if (tid < 16 * NT) {
      float m = sm.m[0][tid], l = sm.l[0][tid];
      for (int w = 1; w < kWaves; ++w) merge_ml(m, l, sm.m[w][tid], sm.l[w][tid]);
      float* st = p.stats + stat_base + ((int64_t)split * kStatRows + tid) * 2;
      st[0] = m;
      st[1] = l;
    }
  }
}

// ---- top-B -------------------------------------------------------------------

// Inclusive prefix sum over the 64 lanes of a wave with DPP moves (no LDS round trips): shifts by
// 1, 2, 4 and 8 lanes within each row of 16 (lanes without a source add 0), then rows 1 and 3 add
// lane 15 of the row below and rows 2 and 3 add lane 31.
__device__ inline uint32_t wave_inclusive_scan(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false);   // row_shr:1
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false);   // row_shr:2
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, false);   // row_shr:4
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, false);   // row_shr:8
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false);   // row_bcast:15
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false);   // row_bcast:31
  return v;
}

// Exclusive prefix sum of x over the workgroup's threads in thread order; total = the sum of all.
// Every wave scans the wave totals itself, so one barrier separates the two levels; the last one
// lets the next call reuse wsum.
__device__ inline uint32_t block_exclusive_scan(uint32_t x, uint32_t* wsum, uint32_t& total) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int kW = kTopkThreads / kWave;
  const uint32_t v = wave_inclusive_scan(x);
  if (lane == kWave - 1) wsum[wave] = v;
  __syncthreads();
  const uint32_t ws = wave_inclusive_scan(lane < kW ? wsum[lane] : 0u);
  const uint32_t below = wave > 0 ? (uint32_t)__builtin_amdgcn_readlane((int)ws, wave - 1) : 0u;
  total = (uint32_t)__builtin_amdgcn_readlane((int)ws, kW - 1);
  __syncthreads();
  return below + v - x;
}

// Add one to bin `d` of a histogram held in `stride` copies (bin d's copy c at d*stride + c; this
// lane adds to copy `copy`).  When every active lane of the wave holds the same digit one lane adds
// the count to copy 0.  Otherwise each lane adds one: an LDS atomic serialises the lanes that meet
// on one word, and the copies spread lanes with equal digits over `stride` words.
__device__ inline void hist_add(uint32_t* hist, uint32_t d, uint32_t stride, uint32_t copy) {
  const uint64_t active = __builtin_amdgcn_read_exec();
  const uint32_t d0 = __builtin_amdgcn_readfirstlane(d);
  const uint64_t same = __builtin_amdgcn_ballot_w64(d == d0);
  if (same == active) {
    if ((uint32_t)__builtin_amdgcn_mbcnt_hi((uint32_t)(active >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)active, 0u)) == 0u)
      atomicAdd(&hist[d0 * stride], (uint32_t)__builtin_popcountll(active));
  } else {
    atomicAdd(&hist[d * stride + copy], 1u);
  }
}

template <int V>
struct IntTag { static constexpr int value = V; };

// Code size matters here: every wave runs each phase once, so a fully unrolled kernel is bound
// by instruction fetch (75 KB of straight-line code measured 39 us).  Only the pooling keeps its
// candidates in registers; it stores them in LDS and every later phase is a short loop over them.
// One workgroup runs the whole (sequence, KV head), so the phases are bound by the CU's own LDS and
// VALU throughput: candidate c belongs to thread c % kTopkThreads (slot e = c / kTopkThreads), so
// a wave's lanes hold consecutive candidates: pooling reads consecutive LDS words (no bank
// conflicts), the keys sit at keys[c], and the ordered compaction ranks candidates by ballots.
__global__ __launch_bounds__(kTopkThreads) void topk_kernel(SelectParams p) {
  constexpr int kTopkWaves = kTopkThreads / kWave;
  constexpr int kPad = 4;                              // -1 words on either side of the staged range
  constexpr int kCells = kMaxPerThread * kTopkWaves;   // (slot, wave) cells of the compaction
  static_assert(2 * kCells <= kHistWords, "compaction counts live in the histogram's space");
  __shared__ float raw_lds[BD_SELECT_MAX_PREFIX + 2 * kPad];   // the pooled range, staged once; then the keys
  __shared__ __align__(16) uint32_t hist[kHistWords];
  __shared__ uint32_t wsum[kTopkWaves];
  __shared__ uint32_t s_digit, s_krem;
  uint32_t* keys = reinterpret_cast<uint32_t*>(raw_lds);
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int pair = blockIdx.x + fetch_select_args(p);
  const int g = pair % p.Hkv, s = pair / p.Hkv;
  const int L = seq_len(p.kv, s);
  const int B = p.budget, W = p.W, ld = p.ld;
  int32_t* idx_row = p.idx_out + (int64_t)pair * ld;

  if (B >= L) {
    for (int t = tid; t < ld; t += kTopkThreads) idx_row[t] = t < L ? t : -1;
    if (g == 0 && tid == 0) p.nsel_out[s] = L;
    return;
  }
  if (g == 0 && tid == 0) p.nsel_out[s] = ld < L ? ld : L;

  // 1. total raw scores (row blocks summed in order), staged in LDS over the prefix [0, N) at
  // raw_lds[kPad + t] and exported when the caller asked for them; each batch of loads is issued
  // before any is summed
  const int N = L - W, K = p.keep, rad = p.pool_kernel / 2;
  float* raw = p.raw ? p.raw + (int64_t)pair * p.max_L : nullptr;
  const float* part = p.raw_part + (int64_t)pair * p.n_rb * p.max_L;
  constexpr int kStageBatch = 16;
  for (int c0 = 0; c0 < L; c0 += kStageBatch * kTopkThreads) {
    float v[kStageBatch];
#pragma unroll
    for (int e = 0; e < kStageBatch; ++e) {
      const int t = c0 + tid + e * kTopkThreads;
      v[e] = t < L ? part[t] : 0.f;
    }
    for (int r = 1; r < p.n_rb; ++r) {
#pragma unroll
      for (int e = 0; e < kStageBatch; ++e) {
        const int t = c0 + tid + e * kTopkThreads;
        if (t < L) v[e] += part[(int64_t)r * p.max_L + t];
      }
    }
#pragma unroll
    for (int e = 0; e < kStageBatch; ++e) {
      const int t = c0 + tid + e * kTopkThreads;
      if (t < N) raw_lds[kPad + t] = v[e];
      if (raw && t < L) raw[t] = v[e];
    }
  }
  if (tid < kPad) { raw_lds[tid] = -1.f; raw_lds[kPad + N + tid] = -1.f; }
  __syncthreads();

  // 2. the candidates: prefix positions [0, N) with max-pooled scores (token level), or the chunks
  // of s positions of the prefix with their scores' sums (TopKChunks, chunk c covering
  // [c*s, min((c+1)*s, N)), summed left to right in fp32).  The top KE of the M candidates are
  // kept.  Scores are >= 0, so their float bits order like their values.
  const int chunk = p.chunk;
  const int M = chunk > 0 ? (N + chunk - 1) / chunk : N;
  int KE = chunk > 0 ? K / chunk : K;
  if (KE > M) KE = M;
  const int E = (M + kTopkThreads - 1) / kTopkThreads;   // slots in use
  const float* rl = raw_lds + kPad;
  uint32_t key[kMaxPerThread];
  if (chunk > 0) {
#pragma unroll
    for (int e = 0; e < kMaxPerThread; ++e) {
      const int c = e * kTopkThreads + tid;
      float sum = 0.f;
      if (e < E && c < M) {
        const int b = c * chunk, n = N - b < chunk ? N - b : chunk;
        for (int j = 0; j < n; ++j) sum += rl[b + j];
      }
      key[e] = e < E && c < M ? __float_as_uint(sum) : 0u;
    }
  } else if (rad <= kPad - 1) {
    // radius <= 3: the -1 words around the range stand in for positions outside it (every
    // pooled score is >= 0), so no bounds checks.  Groups of 8 slots, all reads of a group issued
    // together; a slot past E reads words inside the array and is masked.
    auto pool = [&](auto rtag) {
      constexpr int R = decltype(rtag)::value;
#pragma unroll
      for (int e0 = 0; e0 < kMaxPerThread; e0 += 8) {
        if (e0 < E) {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int e = e0 + j, c = e * kTopkThreads + tid;
            float m = rl[c];
#pragma unroll
            for (int d = 1; d <= R; ++d) m = fmaxf(m, fmaxf(rl[c - d], rl[c + d]));
            key[e] = e < E && c < N ? __float_as_uint(m) : 0u;
          }
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j) key[e0 + j] = 0u;
        }
      }
    };
    if (rad == 3) pool(IntTag<3>{});
    else if (rad == 2) pool(IntTag<2>{});
    else if (rad == 1) pool(IntTag<1>{});
    else pool(IntTag<0>{});
  } else {
    auto raw_at = [&](int t) { return t >= 0 && t < N ? rl[t] : -1.f; };
    float m[kMaxPerThread];
#pragma unroll
    for (int e = 0; e < kMaxPerThread; ++e) m[e] = -1.f;
    for (int d = -rad; d <= rad; ++d) {
#pragma unroll
      for (int e = 0; e < kMaxPerThread; ++e)
        if (e < E) m[e] = fmaxf(m[e], raw_at(e * kTopkThreads + tid + d));
    }
#pragma unroll
    for (int e = 0; e < kMaxPerThread; ++e)
      key[e] = e < E && e * kTopkThreads + tid < N ? __float_as_uint(m[e]) : 0u;
  }
  __syncthreads();                            // every raw value read: the LDS now holds the keys
#pragma unroll
  for (int e = 0; e < kMaxPerThread; ++e)
    if (e < E) keys[e * kTopkThreads + tid] = key[e];
  __syncthreads();
  // Keys in batches of kBatch slots, every read issued before the first is used (an LDS atomic or a
  // ballot between a read and the next would otherwise wait for the LDS round trip each slot).
  // Slots past E read slot E-1 again: the caller's c < M test rejects them.
  constexpr int kBatch = 8;
  auto load_keys = [&](uint32_t (&k)[kBatch], int e0) {
#pragma unroll
    for (int j = 0; j < kBatch; ++j) k[j] = keys[(e0 + j < E ? e0 + j : E - 1) * kTopkThreads + tid];
  };

  // 3. radix select of the KE-th largest key over digits of 8, 11 and 12 bits: the exponent, then
  // the mantissa's top 11 and low 12 bits (the sign bit is always clear); krem = how many keys
  // equal to it are taken.  Most scores share a few exponents and their neighbours share leading
  // mantissa bits, so lane l adds to copy l % 16 (exponent) or l % 2 (top mantissa bits) of the
  // histogram: with one copy of a 12-bit first digit about 18 lanes of a wave met on one word and
  // the serialised atomics took 5 us of the kernel.
  uint32_t prefix = 0, pmask = 0, krem = (uint32_t)KE;
  if (KE > 0) {
    for (int pass = 0; pass < kDigits; ++pass) {
      const int bits = digit_bits(pass), shift = digit_shift(pass);
      const uint32_t ncopy = (uint32_t)digit_copies(pass);
      const uint32_t copy = (uint32_t)lane & (ncopy - 1u);
      const uint32_t nb = 1u << bits, dm = nb - 1;
      for (int i = tid; i < (int)(nb * ncopy); i += kTopkThreads) hist[i] = 0;
      __syncthreads();
      for (int e0 = 0; e0 < E; e0 += kBatch) {
        uint32_t k[kBatch];
        load_keys(k, e0);
#pragma unroll
        for (int j = 0; j < kBatch; ++j)
          if ((e0 + j) * kTopkThreads + tid < M && (k[j] & pmask) == prefix)
            hist_add(hist, (k[j] >> shift) & dm, ncopy, copy);
      }
      __syncthreads();
      // thread tid owns digits nb-1 - (per*tid + q): a block scan counts the keys above them
      constexpr int kMaxPer = kHistWords / kTopkThreads;
      const int per = (int)nb >= kTopkThreads ? (int)nb / kTopkThreads : 1;
      uint32_t h[kMaxPer], c = 0;
#pragma unroll
      for (int q = 0; q < kMaxPer; ++q) {
        const uint32_t x = (uint32_t)(per * tid + q), d = nb - 1 - x;
        h[q] = 0;
        if (q < per && x < nb) {
          if (ncopy >= 4) {
            const uint4* w = reinterpret_cast<const uint4*>(hist + d * ncopy);
            for (uint32_t i = 0; i < ncopy / 4; ++i) { const uint4 v = w[i]; h[q] += v.x + v.y + v.z + v.w; }
          } else if (ncopy == 2) {
            const uint2 v = *reinterpret_cast<const uint2*>(hist + d * 2);
            h[q] = v.x + v.y;
          } else {
            h[q] = hist[d];
          }
        }
        c += h[q];
      }
      uint32_t tot;
      uint32_t a = block_exclusive_scan(c, wsum, tot);
#pragma unroll
      for (int q = 0; q < kMaxPer; ++q) {
        if (q < per && a < krem && krem <= a + h[q]) { s_digit = nb - 1 - (uint32_t)(per * tid + q); s_krem = krem - a; }
        a += h[q];
      }
      __syncthreads();
      prefix |= s_digit << shift;
      pmask |= dm << shift;
      krem = s_krem;
      __syncthreads();
    }
  }

  // 4. ordered compaction: all candidates above the threshold, the first krem equal to it, in
  // ascending order.  Cell (e, wave) holds candidates e*kTopkThreads + 64*wave + [0, 64): ballots
  // count each cell's keys above and equal to the threshold, two scans over the cells in candidate
  // order give each cell its first equal key's rank and its first output slot, and a lane adds the
  // ballot's lanes below it.  A candidate contributes its positions (one, or its chunk's: every
  // chunk but the last has s of them, so a taken candidate's first slot is its rank times s).
  uint32_t* c_eq = hist;                      // per cell: equal keys, then equal keys before it
  uint32_t* c_gt = hist + kCells;             // per cell: keys above, then output slots before it
  const uint64_t below = (1ull << lane) - 1ull;
  const bool any = KE > 0;
  for (int e0 = 0; e0 < E; e0 += kBatch) {
    uint32_t k[kBatch];
    load_keys(k, e0);
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int e = e0 + j, c = e * kTopkThreads + tid;
      const uint64_t beq = __builtin_amdgcn_ballot_w64(any && c < M && k[j] == prefix);
      const uint64_t bgt = __builtin_amdgcn_ballot_w64(any && c < M && k[j] > prefix);
      if (lane == 0 && e < E) {
        c_eq[e * kTopkWaves + wave] = (uint32_t)__builtin_popcountll(beq);
        c_gt[e * kTopkWaves + wave] = (uint32_t)__builtin_popcountll(bgt);
      }
    }
  }
  __syncthreads();
  const int ncell = E * kTopkWaves;
  const uint32_t n_eq = tid < ncell ? c_eq[tid] : 0u, n_gt = tid < ncell ? c_gt[tid] : 0u;
  // One scan of both counts packed as equal << 16 | above (each sum is at most 32768).  The equal
  // keys are taken in candidate order until krem of them are, so min(krem, equal keys before) of
  // them lie in earlier cells.
  uint32_t tot;
  const uint32_t before = block_exclusive_scan(n_eq << 16 | n_gt, wsum, tot);
  const uint32_t eq_before = before >> 16, take_before = (before & 0xFFFFu) + min(krem, eq_before);
  const int taken = (int)((tot & 0xFFFFu) + min(krem, tot >> 16));   // candidates kept
  // Prefix positions kept: unit per taken candidate, less the missing positions of a short last
  // chunk when it is taken (all other equal keys precede it, so an equal last key is taken only
  // when every equal key is).  The window and the unused slots are written first.
  const int unit = chunk > 0 ? chunk : 1;
  int kept = taken * unit;
  if (chunk > 0 && M > 0) {
    const uint32_t kl = keys[M - 1];
    if (any && (kl > prefix || (kl == prefix && krem == tot >> 16))) kept -= unit - (N - (M - 1) * chunk);
  }
  if (kept > K) kept = K;
  for (int i = tid; i < W; i += kTopkThreads) idx_row[kept + i] = N + i;
  for (int i = kept + W + tid; i < ld; i += kTopkThreads) idx_row[i] = -1;   // unused slots
  if (tid < ncell) { c_eq[tid] = eq_before; c_gt[tid] = take_before; }
  __syncthreads();
  for (int e0 = 0; e0 < E; e0 += kBatch) {
    uint32_t k[kBatch], eqb[kBatch], tkb[kBatch];
    load_keys(k, e0);
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int cell = (e0 + j < E ? e0 + j : E - 1) * kTopkWaves + wave;
      eqb[j] = c_eq[cell];
      tkb[j] = c_gt[cell];
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int c = (e0 + j) * kTopkThreads + tid;
      const bool isq = any && c < M && k[j] == prefix;
      const uint64_t beq = __builtin_amdgcn_ballot_w64(isq);
      const bool take = (any && c < M && k[j] > prefix) ||
                        (isq && eqb[j] + (uint32_t)__builtin_popcountll(beq & below) < krem);
      const uint64_t bt = __builtin_amdgcn_ballot_w64(take);
      if (take) {
        const int off = ((int)tkb[j] + __builtin_popcountll(bt & below)) * unit;
        if (chunk == 0) {
          if (off < K) idx_row[off] = c;      // guard: never write past the K prefix slots
        } else {
          const int b = c * chunk, n = N - b < chunk ? N - b : chunk;
          for (int i = 0; i < n; ++i)
            if (off + i < K) idx_row[off + i] = b + i;
        }
      }
    }
  }
}

template <int NT, bool PAGED>
hipError_t launch_scores(const SelectParams& p, int nblocks, hipStream_t stream) {
  if (!p.lse_win) {
    hipLaunchKernelGGL((score_kernel<NT, PAGED, 1>), dim3(nblocks), dim3(kThreads), 0, stream, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((score_kernel<NT, PAGED, 2>), dim3(nblocks), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

int select_nt(int R) {
  const int tiles = (R + 15) / 16;
  return tiles <= 1 ? 1 : tiles <= 2 ? 2 : tiles <= 4 ? 4 : 8;
}

}  // namespace

SelectPlan plan_select(int S, int Hkv, int Hq, int W, int max_L, bool paged, int page_size) {
  SelectPlan pl;
  const int G = Hq / Hkv;
  const int R = W * G;
  const int nt = select_nt(R);
  pl.n_rb = (R + 16 * nt - 1) / (16 * nt);
  const int64_t units = (int64_t)S * Hkv * pl.n_rb;
  const int64_t per_block = (units * max_L + kTargetBlocks - 1) / kTargetBlocks;
  constexpr int64_t kStep = kWaves * kTile;
  int64_t kps = (per_block + kStep - 1) / kStep * kStep;
  const int64_t cap = ((int64_t)max_L + kStep - 1) / kStep * kStep;
  if (kps > cap) kps = cap;
  // a paged split's table holds kSlotCap entries: one per key, or one per page when pages hold whole
  // 16-key sub-tiles (kps keys span at most kps / page_size + 2 pages); keys below 2^26 keep the
  // kernel's page division exact
  pl.page_arith = paged && page_size > 0 && page_size % 16 == 0 && max_L <= (1 << 26) - 64;
  const int64_t paged_cap = pl.page_arith ? ((int64_t)(kSlotCap - 2) * page_size) / kStep * kStep : kMaxPagedKeys;
  if (paged && kps > paged_cap) kps = paged_cap;
  if (kps < kStep) kps = kStep;
  pl.kps = (int)kps;
  pl.nsplit = max_L > 0 ? (int)((max_L + kps - 1) / kps) : 1;
  pl.stats_bytes = align256(sizeof(float) * (size_t)units * pl.nsplit * kStatRows * 2);
  pl.raw_part_bytes = align256(sizeof(float) * (size_t)units * max_L);
  pl.ws_bytes = BD_WS_COUNTER_BYTES + pl.stats_bytes + pl.raw_part_bytes;
  return pl;
}

hipError_t launch_select(const SelectParams& p, bool paged, hipStream_t stream) {
  const int nt = select_nt(p.R);
  const int nblocks = p.S * p.Hkv * p.n_rb * p.nsplit;
  hipError_t e = hipSuccess;
  switch (nt) {
    case 1: e = paged ? launch_scores<1, true>(p, nblocks, stream) : launch_scores<1, false>(p, nblocks, stream); break;
    case 2: e = paged ? launch_scores<2, true>(p, nblocks, stream) : launch_scores<2, false>(p, nblocks, stream); break;
    case 4: e = paged ? launch_scores<4, true>(p, nblocks, stream) : launch_scores<4, false>(p, nblocks, stream); break;
    default: e = paged ? launch_scores<8, true>(p, nblocks, stream) : launch_scores<8, false>(p, nblocks, stream); break;
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(topk_kernel, dim3(p.S * p.Hkv), dim3(kTopkThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace bd
