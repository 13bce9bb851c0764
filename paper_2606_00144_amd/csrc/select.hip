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
//      blocks, max-pools the prefix, finds the (B-W)-th largest pooled score
//      with a 4 x 8-bit radix select over the float bit patterns (scores are
//      non-negative, so the bits order like the values), and compacts the
//      chosen positions in ascending order; ties at the threshold take the
//      lowest positions, then the window is appended.
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
constexpr int kRadixBins0 = 4096;               // bins of the first radix digit (12 bits)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kSlack = 8.f;                    // lazy-rescale headroom of the pass-1 sums, log2 units

__device__ inline void merge_ml(float& m, float& l, float m2, float l2) {
  const float M = fmaxf(m, m2);
  if (M == -INFINITY) { m = M; l = 0.f; return; }
  l = l * exp2f(m - M) + l2 * exp2f(m2 - M);
  m = M;
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
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
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
  if constexpr (PAGED) {
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

  // 16 keys x 16*NT rows of one sub-tile; keys tb .. tb+3 belong to this lane.  `dirty` is a
  // compile-time flag: a runtime one was if-converted, and every tile paid the mask (a compare, a
  // select and a mask merge per score: a third of the loop's VALU instructions).
  auto sub_step = [&](const u32x4 (&kr)[4], int tb, auto dirty_tag) {
    constexpr bool dirty = decltype(dirty_tag)::value;
    f32x4 acc[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      f32x4 a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < 4; ++j) a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kr[j]), qop[nt][j], a, 0, 0, 0);
      acc[nt] = a;
    }
    if constexpr (dirty) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = tb + i;
          if (!(t < k1 && t <= rowpos[nt])) acc[nt][i] = -INFINITY;
        }
    }
    if constexpr (PASS == 1) {
      // per-lane running sum with a lazily raised reference: weights stay <= 2^kSlack.  The check
      // compares raw logits with a per-row threshold, and the raise is a wave-uniform branch (the
      // common tile pays two max and one compare per row tile, no exponential)
      float mx[NT];
      bool raise = false;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        mx[nt] = fmaxf(fmaxf(acc[nt][0], acc[nt][1]), fmaxf(acc[nt][2], acc[nt][3]));
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
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) rl[nt] += __builtin_amdgcn_exp2f(fmaf(acc[nt][i], p.scale_log2, -rm[nt]));
    } else {
      float col[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) col[i] += __builtin_amdgcn_exp2f(fmaf(acc[nt][i], p.scale_log2, -lse2[nt]));
#pragma unroll
      for (int i = 0; i < 4; ++i) col[i] = sum16(col[i]);
      if (lr < 4) {
        const float v = lr == 0 ? col[0] : lr == 1 ? col[1] : lr == 2 ? col[2] : col[3];
        const int t = tb + lr;
        if (t < k1) raw_part[t] = v;
      }
    }
  };

  if (wave < ntiles) {
    const uint32_t ring_lds = lds_addr(sm.ring[wave][0]);
    const uint32_t roff_lds = lds_addr(sm.roff);
    const uint32_t base16 = PAGED ? 0u : (uint32_t)(((int64_t)s * p.kv.stride_seq + (int64_t)g * p.kv.stride_head) >> 3);
    const uint32_t tok16 = (uint32_t)(p.kv.stride_tok >> 3);
    auto issue = [&](int tile, int slot) {
      uint32_t r[2];
      if constexpr (PAGED) {
        read_krows(r, roff_lds, kTile * tile, lane);
      } else if (tile >= ntiles) {
        r[0] = r[1] = 0u;                  // padding: row 0, a safe, cache-resident address
      } else {
        const uint32_t r0 = base16 + (uint32_t)(k0 + kTile * tile) * tok16;
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
      const int tb = k0 + kTile * it + 4 * lg;
      sub_step(kt[0], tb, dirty_tag);
      sub_step(kt[1], tb + 16, dirty_tag);
      ++j;
      return it + kWaves >= ntiles;
    };
    // a wave's tiles increase, so its mask-free ones come first
    bool last = false;
    while (!last && wave + kWaves * j < first_dirty) last = step(std::integral_constant<bool, false>{});
    while (!last) last = step(std::integral_constant<bool, true>{});
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

__device__ inline int block_exclusive_scan(int x, int* wsum, int& total) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int kW = kTopkThreads / kWave;
  int v = x;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int y = __shfl_up(v, o);
    if (lane >= o) v += y;
  }
  if (lane == kWave - 1) wsum[wave] = v;
  __syncthreads();
  if (wave == 0) {
    int w = lane < kW ? wsum[lane] : 0;
#pragma unroll
    for (int o = 1; o < kW; o <<= 1) {
      const int y = __shfl_up(w, o);
      if (lane >= o) w += y;
    }
    if (lane < kW) wsum[lane] = w;
  }
  __syncthreads();
  const int before = (wave > 0 ? wsum[wave - 1] : 0) + v - x;
  total = wsum[kW - 1];
  __syncthreads();
  return before;
}

// Add one to bin `d` of the histogram.  When every active lane of the wave holds the same digit
// (the common case for the leading digits, which the scores mostly share) one lane adds the count,
// so the LDS atomics do not serialise on a single bin.
__device__ inline void hist_add(uint32_t* hist, uint32_t d) {
  const uint64_t active = __builtin_amdgcn_read_exec();
  const uint32_t d0 = __builtin_amdgcn_readfirstlane(d);
  const uint64_t same = __builtin_amdgcn_ballot_w64(d == d0);
  if (same == active) {
    if ((uint32_t)__builtin_amdgcn_mbcnt_hi((uint32_t)(active >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)active, 0u)) == 0u)
      atomicAdd(&hist[d0], (uint32_t)__builtin_popcountll(active));
  } else {
    atomicAdd(&hist[d], 1u);
  }
}

template <int V>
struct IntTag { static constexpr int value = V; };

// Code size matters here: every wave runs each phase once, so a fully unrolled kernel is bound
// by instruction fetch (75 KB of straight-line code measured 39 us).  Only the pooling keeps its
// candidates in registers; it stores them in LDS, striped (candidate e of thread t at
// e*kTopkThreads + t, conflict-free), and every later phase is a short loop over them.
__global__ __launch_bounds__(kTopkThreads) void topk_kernel(SelectParams p) {
  constexpr int kTopkWaves = kTopkThreads / kWave;
  __shared__ float raw_lds[BD_SELECT_MAX_PREFIX];     // the pooled range, staged once; then the keys
  __shared__ uint32_t hist[kRadixBins0];
  __shared__ int wsum[kTopkWaves];
  __shared__ uint32_t s_digit, s_krem;
  uint32_t* keys = reinterpret_cast<uint32_t*>(raw_lds);
  const int tid = threadIdx.x;
  const int pair = blockIdx.x;
  const int g = pair % p.Hkv, s = pair / p.Hkv;
  const int L = seq_len(p.kv, s);
  const int B = p.budget, W = p.W;
  int32_t* idx_row = p.idx_out + (int64_t)pair * B;

  if (B >= L) {
    for (int t = tid; t < B; t += kTopkThreads) idx_row[t] = t < L ? t : -1;
    if (g == 0 && tid == 0) p.nsel_out[s] = L;
    return;
  }
  if (g == 0 && tid == 0) p.nsel_out[s] = B;

  // 1. total raw scores (row blocks summed in order), staged in LDS over the prefix [0, N) and
  // exported when the caller asked for them; each batch of loads is issued before any is summed
  const int N = L - W, K = B - W, rad = p.pool_kernel / 2;
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
      if (t < N) raw_lds[t] = v[e];
      if (raw && t < L) raw[t] = v[e];
    }
  }
  __syncthreads();

  // 2. the candidates: prefix positions [0, N) with max-pooled scores (token level), or the chunks
  // of s positions of the prefix with their scores' sums (TopKChunks, chunk c covering
  // [c*s, min((c+1)*s, N)), summed left to right in fp32).  This thread owns candidates
  // [t0, t0 + E); the top KE of the M candidates are kept.  Scores are >= 0, so their float bits
  // order like their values.
  const int chunk = p.chunk;
  const int M = chunk > 0 ? (N + chunk - 1) / chunk : N;
  int KE = chunk > 0 ? K / chunk : K;
  if (KE > M) KE = M;
  const int E = (M + kTopkThreads - 1) / kTopkThreads;
  const int t0 = tid * E;
  uint32_t key[kMaxPerThread];
  auto raw_at = [&](int t) { return t >= 0 && t < N ? raw_lds[t] : -1.f; };
  if (chunk > 0) {
#pragma unroll
    for (int e = 0; e < kMaxPerThread; ++e) {
      const int c = t0 + e;
      float sum = 0.f;
      if (e < E && c < M) {
        const int b = c * chunk, n = N - b < chunk ? N - b : chunk;
        for (int j = 0; j < n; ++j) sum += raw_lds[b + j];
      }
      key[e] = e < E && c < M ? __float_as_uint(sum) : 0u;
    }
  } else if (rad <= 3) {
    // radius <= 3: the thread's window of raw values in registers (every load issued before any
    // max), one code path for every such radius (maxima past the radius are masked)
    float w[kMaxPerThread + 6];
#pragma unroll
    for (int i = 0; i < kMaxPerThread + 6; ++i) w[i] = i < E + 6 ? raw_at(t0 - 3 + i) : -1.f;
#pragma unroll
    for (int e = 0; e < kMaxPerThread; ++e) {
      float m = w[e + 3];
#pragma unroll
      for (int d = 1; d <= 3; ++d) m = fmaxf(m, d <= rad ? fmaxf(w[e + 3 - d], w[e + 3 + d]) : -1.f);
      key[e] = e < E && t0 + e < N ? __float_as_uint(m) : 0u;   // m >= 0: bits order like values
    }
  } else {
    float m[kMaxPerThread];
#pragma unroll
    for (int e = 0; e < kMaxPerThread; ++e) m[e] = -1.f;
    for (int d = -rad; d <= rad; ++d) {
#pragma unroll
      for (int e = 0; e < kMaxPerThread; ++e)
        if (e < E) m[e] = fmaxf(m[e], raw_at(t0 + e + d));
    }
#pragma unroll
    for (int e = 0; e < kMaxPerThread; ++e) key[e] = e < E && t0 + e < N ? __float_as_uint(m[e]) : 0u;
  }
  __syncthreads();                            // every raw value read: the LDS now holds the keys
#pragma unroll
  for (int e = 0; e < kMaxPerThread; ++e)
    if (e < E) keys[e * kTopkThreads + tid] = key[e];
  __syncthreads();
  auto key_at = [&](int e) { return keys[e * kTopkThreads + tid]; };

  // 3. radix select of the KE-th largest key over digits of 12, 10 and 10 bits; krem = how many keys
  // equal to it are taken.  A 12-bit first digit (sign, exponent, 3 mantissa bits) spreads each
  // binade over 8 bins: with 8 bits the scores' few exponents piled thousands of LDS atomics onto a
  // handful of bins.
  uint32_t prefix = 0, pmask = 0, krem = (uint32_t)KE;
  if (KE > 0) {
    for (int pass = 0; pass < 3; ++pass) {
      const int bits = pass == 0 ? 12 : 10, shift = pass == 0 ? 20 : (pass == 1 ? 10 : 0);
      const uint32_t nb = 1u << bits, dm = nb - 1;
      for (int i = tid; i < (int)nb; i += kTopkThreads) hist[i] = 0;
      __syncthreads();
#pragma unroll 4
      for (int e = 0; e < E; ++e) {
        const uint32_t k = key_at(e);
        if (t0 + e < M && (k & pmask) == prefix) hist_add(hist, (k >> shift) & dm);
      }
      __syncthreads();
      // thread tid owns digits nb-1 - (per*tid + q): a block scan counts the keys above them
      const int per = (int)nb / kTopkThreads;
      uint32_t c = 0;
      for (int q = 0; q < per; ++q) c += hist[nb - 1 - (per * tid + q)];
      int tot;
      uint32_t a = (uint32_t)block_exclusive_scan((int)c, wsum, tot);
      for (int q = 0; q < per; ++q) {
        const uint32_t h = hist[nb - 1 - (per * tid + q)];
        if (a < krem && krem <= a + h) { s_digit = nb - 1 - (uint32_t)(per * tid + q); s_krem = krem - a; }
        a += h;
      }
      __syncthreads();
      prefix |= s_digit << shift;
      pmask |= dm << shift;
      krem = s_krem;
      __syncthreads();
    }
  }

  // 4. ordered compaction: all candidates above the threshold, the first krem equal to it; a
  // candidate contributes its positions (one, or its chunk's), in ascending order
  auto positions = [&](int c) {
    if (chunk == 0) return 1;
    const int b = c * chunk;
    return N - b < chunk ? N - b : chunk;
  };
  const int Ev = KE > 0 ? (M - t0 < E ? (M - t0 > 0 ? M - t0 : 0) : E) : 0;   // this thread's candidates
  int eq = 0;
#pragma unroll 4
  for (int e = 0; e < Ev; ++e) eq += key_at(e) == prefix;
  int tot;
  const int eq_before = block_exclusive_scan(eq, wsum, tot);
  int take_eq = (int)krem - eq_before;
  take_eq = take_eq < 0 ? 0 : (take_eq > eq ? eq : take_eq);
  int mine = 0, seen = 0;
#pragma unroll 4
  for (int e = 0; e < Ev; ++e) {
    const uint32_t k = key_at(e);
    const bool isq = k == prefix;
    if (k > prefix || (isq && seen < take_eq)) mine += positions(t0 + e);
    seen += isq;
  }
  int kept;                                   // prefix positions kept: K (token level), <= K (chunks)
  int off = block_exclusive_scan(mine, wsum, kept);
  seen = 0;
  for (int e = 0; e < Ev; ++e) {
    const int c = t0 + e;
    const uint32_t k = key_at(e);
    const bool isq = k == prefix;
    if (k > prefix || (isq && seen < take_eq)) {
      const int n = positions(c), b = chunk > 0 ? c * chunk : c;
      for (int j = 0; j < n; ++j, ++off)
        if (off < K) idx_row[off] = b + j;    // guard: never write past the B - W prefix slots
    }
    seen += isq;
  }
  if (kept > K) kept = K;
  for (int i = tid; i < W; i += kTopkThreads) idx_row[kept + i] = N + i;
  for (int i = kept + W + tid; i < B; i += kTopkThreads) idx_row[i] = -1;   // chunk mode: unused slots
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

SelectPlan plan_select(int S, int Hkv, int Hq, int W, int max_L, bool paged) {
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
  if (paged && kps > kMaxPagedKeys) kps = kMaxPagedKeys;
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
