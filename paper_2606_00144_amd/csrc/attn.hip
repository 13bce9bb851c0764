// Attention of a small block of query rows over a KV range, on gfx950 MFMA.
//
// One kernel serves three operations:
//   - drafter decode over the selected entries K_S^sp(B) (Eq. 2),
//   - verifier attention at the gamma+1 draft positions over the full cache (Eq. 1),
//   - the continuation block under several sparse views and the full cache (Alg. 1).
// Each is "R query rows of one KV head against a key set", where the key set is
// either a gathered index list (a sparse view) or the causal prefix (full).
//
// Work decomposition.  A unit is (key source, sequence s, KV head g, row block
// rb of up to 32 rows).  Its keys are cut into splits; one 256-thread
// workgroup (4 waves) handles one (unit, split), each wave taking every 4th
// 32-key tile.  A wave keeps an online-softmax state (running max, sum and
// output) per row; the 4 waves merge through LDS; the splits of a unit merge
// in the last workgroup to finish (atomic counter), in split order, so the
// result is bitwise reproducible.
//
// MFMA layout (v_mfma_f32_16x16x32_bf16; A is 16x32, B is 32x16, D is 16x16;
// lane l feeds row/col l%16 and a group of 8 k-slots chosen by l/16; D
// element (4*(l/16)+i, l%16) sits in lane l, register i):
//   scores   S^T[key][row] = K[key][:] . Q[row][:]   A = K tile, B = Q^T
//   output   O^T[d][row]  += V^T[d][key] . P^T[key][row]
// With keys on the M side, lane l ends up holding the probabilities of query
// row l%16 for 8 keys, which are exactly the k-slots it must feed as the B
// operand of the second product: P never leaves registers.  The softmax
// statistics of row l%16 also live in lane l.  V^T needs each lane to hold
// 8 keys of one d; each lane loads 16 contiguous bytes (8 d values) of 8 key
// rows (4 full rows per load instruction across the wave, fully coalesced)
// and transposes the 8x8 bf16 block in registers with byte permutes.
// The head dimension is contracted in a lane-group-major order (lane group
// l/16 owns d in [32*(l/16), 32*(l/16)+32)), so each lane reads 64 contiguous
// bytes of a key row; the order of a contraction does not change its value.

#include "bd_common.hpp"
#include "bd_kernels.hpp"
#include "attn_tile.hpp"

namespace bd {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * kWave;
constexpr int kTile = 32;                      // keys per wave iteration
constexpr int64_t kTargetBlocks = 256;         // workgroups per launch the splits aim for (one per CU)
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kSlack = 8.f;                  // lazy-rescale headroom, log2 units

template <int NT>
struct RowBlock {
  static constexpr int kRows = 16 * NT;
  // floats of one partial record: per row (m, l, lx, unused), then the unnormalised outputs
  static constexpr int kRec = kRows * (4 + kD);
};

// Key slots of one split: row offset (16-byte units) and position of every
// key, resolved once per workgroup (idx gather, page-table lookup, bounds) so
// that the streaming loop issues only unconditional loads.  kAhead extra tiles
// per wave of padding slots (position -1, offset 0: a safe address) let every
// wave prefetch past its last tile without a branch.
// Each wave streams its tiles through kRing LDS slots with direct-to-LDS
// loads (global_load_lds_dwordx4), which need no registers while in flight: a
// tile is copied to registers just before its step and its slot is refilled at
// once, so kRing tiles stay in flight during every step.
constexpr int kRing = 2;
constexpr int kTileLoads = 16;                  // 16-byte loads per lane per tile: K 8, V 8
constexpr int kTileBytes = kTileLoads * kWave * 16;
constexpr int kMaxAhead = kRing;
constexpr int kSlotCap = kMaxSplitKeys + kMaxAhead * kWaves * kTile;

// LDS scratch of one workgroup: the slot table while streaming, the per-wave
// partial outputs while merging (separated by a barrier).
template <int NT>
struct AttnSmem {
  union {
    struct {
      alignas(16) int32_t roff[kSlotCap];
      alignas(16) int32_t tpos[kSlotCap];
      alignas(16) uint8_t ring[kWaves][kRing][kTileBytes];   // per-wave tile slots filled by DMA
    } slots;
    struct {
      alignas(16) float o[kWaves][16 * NT][kD + 4]; // per-wave unnormalised outputs (rows padded: the
                                                    // 16 rows a store instruction writes hit distinct banks)
      float m[kWaves][16 * NT];
      float l[kWaves][16 * NT];
      float lx[kWaves][16 * NT];
    } merge;
  } u;
  int32_t first_dirty[kWaves];   // per wave: first tile of its table chunks that needs the mask
  int32_t last;
};

template <int NT, bool PAGED>
struct TileRegs {
  u32x4 k[2][4];     // [key subtile][k-step]: 16 keys x 64 B per lane group
  u32x4 v[8];        // 8 key rows x 16 B
  u32x4 tp[2];       // positions of the 8 score slots (-1 = absent), slot i in tp[i/4][i%4]
};

// Row offsets (16-byte units) of the 10 key rows a lane loads for one tile:
// K rows slot0+lr and slot0+16+lr, V rows slot0 + 16h + 4*(lane/16) + 0..3.
struct TileRows {
  uint32_t k[2];
  u32x4 v[2];
};

// Read a tile's row offsets from the LDS slot table: loads and their wait in one asm statement.
__device__ inline void read_rows(TileRows& A, uint32_t roff_lds, int slot0, int lane) {
  const int lg = lane >> 4, lr = lane & 15;
  const uint32_t ak = roff_lds + 4 * (slot0 + lr);
  const uint32_t av = roff_lds + 4 * (slot0 + 4 * lg);
  asm volatile(
      "ds_read_b32 %0, %4\n"
      "ds_read_b32 %1, %4 offset:64\n"
      "ds_read_b128 %2, %5\n"
      "ds_read_b128 %3, %5 offset:64\n"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(A.k[0]), "=&v"(A.k[1]), "=&v"(A.v[0]), "=&v"(A.v[1])
      : "v"(ak), "v"(av));
}

// Copy the landed tile in LDS slot `src` into registers and read the row offsets of the
// tile to prefetch next, all in one asm statement ending in its own wait.
template <int NT, bool PAGED>
__device__ inline void read_tile_and_rows(TileRegs<NT, PAGED>& T, TileRows& A, uint32_t src, uint32_t tpos_lds,
                                          int slot0, uint32_t roff_lds, int next0, int lane) {
  const int lg = lane >> 4, lr = lane & 15;
  const uint32_t at = src + 16 * lane;
  const uint32_t ap = tpos_lds + 4 * (slot0 + 4 * lg);
  const uint32_t ak = roff_lds + 4 * (next0 + lr);
  const uint32_t av = roff_lds + 4 * (next0 + 4 * lg);
  asm volatile(
      "ds_read_b128 %0, %22\n"
      "ds_read_b128 %1, %22 offset:1024\n"
      "ds_read_b128 %2, %22 offset:2048\n"
      "ds_read_b128 %3, %22 offset:3072\n"
      "ds_read_b128 %4, %22 offset:4096\n"
      "ds_read_b128 %5, %22 offset:5120\n"
      "ds_read_b128 %6, %22 offset:6144\n"
      "ds_read_b128 %7, %22 offset:7168\n"
      "ds_read_b128 %8, %22 offset:8192\n"
      "ds_read_b128 %9, %22 offset:9216\n"
      "ds_read_b128 %10, %22 offset:10240\n"
      "ds_read_b128 %11, %22 offset:11264\n"
      "ds_read_b128 %12, %22 offset:12288\n"
      "ds_read_b128 %13, %22 offset:13312\n"
      "ds_read_b128 %14, %22 offset:14336\n"
      "ds_read_b128 %15, %22 offset:15360\n"
      "ds_read_b128 %16, %23\n"
      "ds_read_b128 %17, %23 offset:64\n"
      "ds_read_b32 %18, %24\n"
      "ds_read_b32 %19, %24 offset:64\n"
      "ds_read_b128 %20, %25\n"
      "ds_read_b128 %21, %25 offset:64\n"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(T.k[0][0]), "=&v"(T.k[0][1]), "=&v"(T.k[0][2]), "=&v"(T.k[0][3]), "=&v"(T.k[1][0]),
        "=&v"(T.k[1][1]), "=&v"(T.k[1][2]), "=&v"(T.k[1][3]), "=&v"(T.v[0]), "=&v"(T.v[1]), "=&v"(T.v[2]),
        "=&v"(T.v[3]), "=&v"(T.v[4]), "=&v"(T.v[5]), "=&v"(T.v[6]), "=&v"(T.v[7]), "=&v"(T.tp[0]), "=&v"(T.tp[1]),
        "=&v"(A.k[0]), "=&v"(A.k[1]), "=&v"(A.v[0]), "=&v"(A.v[1])
      : "v"(at), "v"(ap), "v"(ak), "v"(av));
}

// Copy the landed tile in LDS slot `src` into registers (keys whose row offsets are computed).
template <int NT, bool PAGED>
__device__ inline void read_tile(TileRegs<NT, PAGED>& T, uint32_t src, int lane) {
  const uint32_t at = src + 16 * lane;
  asm volatile(
      "ds_read_b128 %0, %16\n"
      "ds_read_b128 %1, %16 offset:1024\n"
      "ds_read_b128 %2, %16 offset:2048\n"
      "ds_read_b128 %3, %16 offset:3072\n"
      "ds_read_b128 %4, %16 offset:4096\n"
      "ds_read_b128 %5, %16 offset:5120\n"
      "ds_read_b128 %6, %16 offset:6144\n"
      "ds_read_b128 %7, %16 offset:7168\n"
      "ds_read_b128 %8, %16 offset:8192\n"
      "ds_read_b128 %9, %16 offset:9216\n"
      "ds_read_b128 %10, %16 offset:10240\n"
      "ds_read_b128 %11, %16 offset:11264\n"
      "ds_read_b128 %12, %16 offset:12288\n"
      "ds_read_b128 %13, %16 offset:13312\n"
      "ds_read_b128 %14, %16 offset:14336\n"
      "ds_read_b128 %15, %16 offset:15360\n"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(T.k[0][0]), "=&v"(T.k[0][1]), "=&v"(T.k[0][2]), "=&v"(T.k[0][3]), "=&v"(T.k[1][0]),
        "=&v"(T.k[1][1]), "=&v"(T.k[1][2]), "=&v"(T.k[1][3]), "=&v"(T.v[0]), "=&v"(T.v[1]), "=&v"(T.v[2]),
        "=&v"(T.v[3]), "=&v"(T.v[4]), "=&v"(T.v[5]), "=&v"(T.v[6]), "=&v"(T.v[7])
      : "v"(at));
}

// Issue the direct-to-LDS loads of a tile into `dst`: load q of a lane lands at
// dst + q*1 KiB + 16*lane (q 0..7: K subtile q/4, k-step q%4; q 8..15: V row slot q-8).
// Row offsets are clamped to the layout's extent (validated on the host), so no
// value can address outside the K/V allocation.  `stream_v`: the V rows are read
// once per call (the full branch of verify) and load non-temporally.  Measured on
// the 16K verify: 100 -> 85 us.  Whole-line V reads gain, while the K reads, each
// line taken in four 32-byte parts by four instructions, lose under the same
// policy.  Gathered lists keep the default: the drafts re-read their entries.
__device__ inline void dma_tile(const KvView& kv, const TileRows& A, uint32_t max_roff, uint8_t* dst, int lane,
                                bool stream_v) {
  const int lg = lane >> 4, lr = lane & 15;
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) {
    const uint32_t ro = A.k[sub] < max_roff ? A.k[sub] : max_roff;
    const uint16_t* kr = kv.k + ((uint64_t)ro << 3) + 32 * lg;
#pragma unroll
    for (int j = 0; j < 4; ++j) dma16(kr + 8 * j, dst + (4 * sub + j) * 1024);
  }
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t ro = A.v[h][i] < max_roff ? A.v[h][i] : max_roff;
      if (stream_v) dma16_nt(kv.v + ((uint64_t)ro << 3) + 8 * lr, dst + (8 + 4 * h + i) * 1024);
      else dma16(kv.v + ((uint64_t)ro << 3) + 8 * lr, dst + (8 + 4 * h + i) * 1024);
    }
}

// V rows already in the tile registers.
template <int NT, bool PAGED>
__device__ inline auto pass_v(const TileRegs<NT, PAGED>& T) {
  return [&T](u32x4 (&v)[8]) {
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = T.v[i];
  };
}

template <int NT>
struct RowState {
  f32x4 o[NT][8];     // O^T[d-tile][row tile]
  f32x4 l[NT];        // row sums of the bf16-rounded weights the PV product uses (normaliser), accumulated
                      // by an MFMA against an all-ones operand: every register holds the row's total
  float m[NT];        // running max (log2 domain), shared by the 4 lane groups
  float lx[NT];       // this lane's keys' sum of the unrounded weights (log-sum-exp only)
};

// One 32-key tile of one wave.  `dirty` (wave-uniform) asks for the visibility mask: only tiles
// at the causal edge, at the ragged end of a split or holding absent entries need it.  `want_lx`
// (uniform) keeps the exact weight sum the log-sum-exp output is computed from.
// `get_v` delivers the tile's V rows (8 x 16 bytes per lane) just before the PV product, so a caller
// may read them from LDS only then; they are transposed here (register i of d-tile dt holds
// d = 32*(l/16) + 8*i + dt).
template <int NT, bool PAGED, class PosFn, class VFn>
__device__ inline void tile_step(RowState<NT>& st, const TileRegs<NT, PAGED>& T, const bf16x8 (&qop)[NT][4],
                                 const int (&rowpos)[NT], float scale_log2, bool dirty, bool want_lx,
                                 PosFn pos_of, VFn get_v) {
  // scores S^T for 32 keys x 16*NT rows (unscaled)
  f32x4 sacc[2][NT];
#pragma unroll
  for (int sub = 0; sub < 2; ++sub)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      f32x4 a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < 4; ++j)
        a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(T.k[sub][j]), qop[nt][j], a, 0, 0, 0);
      sacc[sub][nt] = a;
    }

  if (dirty) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int tpos = pos_of(i);   // position of score slot i, -1 when absent
        if (!(tpos >= 0 && tpos <= rowpos[nt])) sacc[i >> 2][nt][i & 3] = -INFINITY;
      }
  }

  // online softmax with a lazily raised reference max: the accumulators are rescaled only when a
  // tile's max exceeds the reference by more than kSlack (log2 units), so weights stay <= 2^kSlack
  // and the common tile costs no rescale.  The rescale branch is taken by the whole wave when any
  // row needs it (rows that do not get factor 1), so it stays a scalar branch.
  float mx[NT];
  bool raise = false;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float v = -INFINITY;
#pragma unroll
    for (int i = 0; i < 8; ++i) v = fmaxf(v, sacc[i >> 2][nt][i & 3]);
    mx[nt] = max_xor32(max_xor16(v)) * scale_log2;    // scale > 0: the max commutes with it
    raise |= mx[nt] > st.m[nt] + kSlack;
  }
  if (__builtin_expect(__builtin_amdgcn_ballot_w64(raise) != 0, 0)) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const bool up = mx[nt] > st.m[nt] + kSlack;
      const float alpha = up ? __builtin_amdgcn_exp2f(st.m[nt] - mx[nt]) : 1.f;   // 0 on the first visible tile
      st.m[nt] = up ? mx[nt] : st.m[nt];
      st.l[nt] *= alpha;
      st.lx[nt] *= alpha;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) st.o[nt][dt] *= alpha;
    }
  }

  const bf16x8 ones = as_bf16x8(u32x4{0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u});
  bf16x8 pop[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const float muse = st.m[nt] == -INFINITY ? 0.f : st.m[nt];
    float pv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) pv[i] = __builtin_amdgcn_exp2f(fmaf(sacc[i >> 2][nt][i & 3], scale_log2, -muse));
    u32x4 pw;
#pragma unroll
    for (int i = 0; i < 4; ++i) pw[i] = pack_bf16x2(pv[2 * i], pv[2 * i + 1]);
    pop[nt] = as_bf16x8(pw);
    if (want_lx) {
      float sx = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) sx += pv[i];
      st.lx[nt] += sx;
    }
    // the normaliser sums exactly the rounded weights the PV product sees
    st.l[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pop[nt], st.l[nt], 0, 0, 0);
  }

  u32x4 vrows[8];
  get_v(vrows);
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) {
    const bf16x8 vt = vt_operand(vrows, dt);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
      st.o[nt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vt, pop[nt], st.o[nt][dt], 0, 0, 0);
  }
}

// Kernel arguments reach the waves through the scalar cache, one 64-byte line per miss, and the
// compiler fetches each where it is first used: a memory round trip apiece, several in a row before
// the first data load and again before the merge.  Naming them all at entry has every line
// requested at once, so the arguments cost one round trip.  The statements touch no memory (so the
// uniform loads after them stay scalar) and return 0, which the caller adds to its block index.
template <bool PAGED>
__device__ inline int fetch_args(const AttnParams& p) {
  int z0, z1, z2;
  asm("s_mov_b32 %0, 0" : "=s"(z0) : "s"(p.kv.k), "s"(p.kv.v), "s"(p.kv.seq_lens), "s"(p.kv.page_table),
      "s"(p.kv.stride_seq), "s"(p.kv.stride_head), "s"(p.kv.stride_tok), "s"(p.kv.stride_page),
      "s"(p.kv.max_seq_len), "s"(p.kv.page_size), "s"(p.kv.max_pages_per_seq), "s"(p.kv.num_pages));
  asm("s_mov_b32 %0, 0" : "=s"(z1) : "s"(z0), "s"(p.q), "s"(p.out_g), "s"(p.out_f), "s"(p.lse_g), "s"(p.lse_f),
      "s"(p.idx), "s"(p.nsel), "s"(p.ld_idx), "s"(p.S), "s"(p.Hkv), "s"(p.Hq), "s"(p.G), "s"(p.nq), "s"(p.R),
      "s"(p.n_rb));
  asm("s_mov_b32 %0, 0" : "=s"(z2) : "s"(z1), "s"(p.nsplit_g), "s"(p.kps_g), "s"(p.nsplit_f), "s"(p.kps_f),
      "s"(p.units_g), "s"(p.nblk_g), "s"(p.nblk), "s"(p.scale_log2), "s"(p.max_roff), "s"(p.part),
      "s"(p.counters));
  if constexpr (PAGED) asm("s_mov_b32 %0, 0" : "=s"(z2) : "s"(z2), "s"(p.page_arith));
  return z2;
}

__device__ inline f32x4 as_f32x4(const u32x4& v) { return __builtin_bit_cast(f32x4, v); }
__device__ inline u32x4 as_u32x4(const f32x4& v) { return __builtin_bit_cast(u32x4, v); }
__device__ inline u32x4 pack_record_bf16(const f32x4& a, const f32x4& b) {
  return u32x4{pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3]), pack_bf16x2(b[0], b[1]), pack_bf16x2(b[2], b[3])};
}
__device__ inline void unpack_record_bf16(const u32x4& w, f32x4& a, f32x4& b) {
  a = f32x4{bf16_lo(w[0]), bf16_hi(w[0]), bf16_lo(w[1]), bf16_hi(w[1])};
  b = f32x4{bf16_lo(w[2]), bf16_hi(w[2]), bf16_lo(w[3]), bf16_hi(w[3])};
}

// Records merged by one batch of loads; units with more splits merge in two levels (TWO_LEVEL, chosen
// per launch when some unit has more than kMergeGroup splits; the one-level merge keeps its own code).
constexpr int kMergeGroup = 8;

template <int NT, bool PAGED, bool TWO_LEVEL>
__global__ __launch_bounds__(kThreads) void attn_kernel(AttnParams p) {
  using RB = RowBlock<NT>;
  __shared__ AttnSmem<NT> sm;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: LDS slot addresses stay scalar
  const int lg = lane >> 4, lr = lane & 15;

  // ---- which (kind, unit, split) this workgroup owns
  const int bid = xcd_remap(blockIdx.x + fetch_args<PAGED>(p), p.nblk);
  const bool gather = bid < p.nblk_g;
  const int local = gather ? bid : bid - p.nblk_g;
  const int nsplit = gather ? p.nsplit_g : p.nsplit_f;
  const int kps = gather ? p.kps_g : p.kps_f;
  // block indices are far below 2^22: float-reciprocal divisions
  const int rest = div_small(local, p.n_rb);
  const int rb = local - rest * p.n_rb;
  const int pair = div_small(rest, nsplit);  // gather: (view, s, g); full: (s, g)
  const int split = rest - pair * nsplit;
  const int vs = div_small(pair, p.Hkv);     // gather: view*S + s; full: s
  const int g = pair - vs * p.Hkv;
  const int view = gather ? div_small(vs, p.S) : 0;
  const int s = vs - view * p.S;
  const int unit = gather ? pair * p.n_rb + rb : p.units_g + pair * p.n_rb + rb;

  // ---- prologue: every load it needs (cache length, entry count, query rows, the split's idx
  // entries) is issued before any of them is used, so they share one memory round trip
  const int L_raw = p.kv.seq_lens[s];
  const int n_raw = *(gather ? p.nsel + vs : p.kv.seq_lens + s);
  const int32_t* idx_row = gather ? p.idx + ((int64_t)vs * p.Hkv + g) * p.ld_idx : nullptr;
  // query rows of this lane: row n = rb*RB + 16*nt + lane%16
  bf16x8 qop[NT][4];
  int qj[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int n = rb * RB::kRows + 16 * nt + lr;
    const bool valid = n < p.R;
    const int jn = div_small(n, p.G);
    const int j = valid ? jn : 0;
    const int h = g * p.G + (valid ? n - jn * p.G : 0);
    qj[nt] = valid ? j : -1;
    const uint16_t* qrow = p.q + (((int64_t)s * p.nq + j) * p.Hq + h) * kD + 32 * lg;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) qop[nt][kk] = as_bf16x8(valid ? load16(qrow + 8 * kk) : u32x4{0u, 0u, 0u, 0u});
  }
  // the causal prefix of a contiguous cache needs no slot table: row offsets are computed.  So are
  // they for the prefix of a paged cache whose pages hold whole 16-key sub-tiles (page_size a
  // multiple of 16, checked on the host), from a table of page offsets: one entry per page, so the
  // split is bounded by kSlotCap pages rather than kSlotCap keys
  const bool arith = !PAGED && !gather;
  const bool page_arith = PAGED && !gather && p.page_arith != 0;
  const int e_begin = split * kps;       // a multiple of kWaves * kTile
  // slot-table entries: the idx loads do not wait for the entry count (every entry of the split
  // below ld_idx lies in the list's row; those past the count are dropped once it has arrived)
  constexpr int kPer = (kSlotCap + kThreads - 1) / kThreads;
  int tv[kPer];
  // page table: the entries of every page the split can touch below max_seq_len (the length is not
  // waited for; pages past it are dropped once it has arrived).  key / page_size is computed as
  // (key / 16) / (page_size / 16), exact for keys below 2^26 (host-checked)
  const int psub = PAGED ? p.kv.page_size >> 4 : 1;
  const float inv_psub = __builtin_amdgcn_rcpf((float)psub);
  const int page0 = page_arith ? div_small(e_begin >> 4, psub, inv_psub) : 0;
  int npg_ld = 0;
  if (page_arith) {
    const int kend = e_begin + kps < p.kv.max_seq_len ? e_begin + kps : p.kv.max_seq_len;
    npg_ld = kend > e_begin ? div_small((kend - 1) >> 4, psub, inv_psub) - page0 + 1 : 0;
    const int32_t* prow = p.kv.page_table + (int64_t)s * p.kv.max_pages_per_seq + page0;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int j = tid + k * kThreads;
      tv[k] = j < npg_ld ? prow[j] : -1;
    }
  } else if (!arith) {
    const int e_lim = gather ? (e_begin + kps < p.ld_idx ? e_begin + kps : p.ld_idx) : e_begin + kps;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int e = e_begin + tid + k * kThreads;
      tv[k] = e < e_lim ? (gather ? idx_row[e] : e) : -1;
    }
  }

  const int L = L_raw < 0 ? 0 : (L_raw > p.kv.max_seq_len ? p.kv.max_seq_len : L_raw);
  const int n_keys = gather ? (n_raw < 0 ? 0 : (n_raw > p.ld_idx ? p.ld_idx : n_raw)) : L;
  int rowpos[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) rowpos[nt] = qj[nt] >= 0 ? L - p.nq + qj[nt] : 0x7FFFFFFF;

  int e_end = e_begin + kps;
  if (e_end > n_keys) e_end = n_keys;

  const int ntiles = e_end > e_begin ? (e_end - e_begin + kTile - 1) / kTile : 0;
  const int nslots = (ntiles + kMaxAhead * kWaves) * kTile;     // <= kSlotCap: padding tiles included
  // a tile needs the visibility mask when one of its slots is absent or lies after the earliest
  // row position of this row block; the first such tile bounds the mask-free ones
  const int minpos = L - p.nq + div_small(rb * RB::kRows, p.G);
  bool page_bad = false;                 // a page the split needs is outside the pool: its keys are absent
  if (page_arith) {
    // page offsets in 16-byte units of head g; -1 marks an entry outside the pool (offsets stay below
    // max_roff < 2^31, host-checked)
    const int npg = e_end > e_begin ? div_small((e_end - 1) >> 4, psub, inv_psub) - page0 + 1 : 0;
    int bad = 0;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int j = tid + k * kThreads;
      if (j < npg_ld) {
        const bool ok = (unsigned)tv[k] < (unsigned)p.kv.num_pages;
        sm.u.slots.roff[j] =
            ok ? (int)(((int64_t)tv[k] * p.kv.stride_page + (int64_t)g * p.kv.stride_head) >> 3) : -1;
        bad |= (j < npg && !ok) ? 1 : 0;
      }
    }
    page_bad = __syncthreads_or(bad) != 0;
  } else if (!arith) {
    // entries past the split's end or outside [0, L) become padding; all page-table loads are
    // issued before any result is used
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int e = e_begin + tid + k * kThreads;
      const int t = e < e_end ? tv[k] : -1;
      tv[k] = (t >= 0 && t < L) ? t : -1;
    }
    int pg[kPer];
    if constexpr (PAGED) {
#pragma unroll
      for (int k = 0; k < kPer; ++k)
        pg[k] = tv[k] >= 0 ? p.kv.page_table[(int64_t)s * p.kv.max_pages_per_seq + tv[k] / p.kv.page_size] : 0;
    }
    // row offsets in 16-byte units: 32-bit products for a contiguous cache (strides are multiples
    // of 8 elements and every offset stays below max_roff < 2^32, both checked on the host)
    const uint32_t base16 = (uint32_t)(((int64_t)s * p.kv.stride_seq + (int64_t)g * p.kv.stride_head) >> 3);
    const uint32_t tok16 = (uint32_t)(p.kv.stride_tok >> 3);
    int first_dirty = 0x7FFFFFFF;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      if (k * kThreads >= nslots) break;     // uniform: the rest of the table is unused
      const int i = tid + k * kThreads;
      bool bad = false;
      if (i < nslots) {
        int t = tv[k];
        uint32_t ro;
        if constexpr (PAGED) {
          const int64_t o = (unsigned)pg[k] < (unsigned)p.kv.num_pages
                                ? (int64_t)pg[k] * p.kv.stride_page + (int64_t)g * p.kv.stride_head +
                                      (int64_t)(t % p.kv.page_size) * p.kv.stride_tok
                                : -1;
          if (t < 0 || o < 0) t = -1;
          ro = t < 0 ? 0u : (uint32_t)(o >> 3);
        } else {
          ro = t < 0 ? 0u : base16 + (uint32_t)t * tok16;
        }
        sm.u.slots.roff[i] = (int)ro;
        sm.u.slots.tpos[i] = t;
        bad = i < ntiles * kTile && (t < 0 || t > minpos);
      }
      // chunk k of this wave is slots k*kThreads + 64*wave .. +63: two tiles, the low 32 ballot bits the first
      const uint64_t mask = __builtin_amdgcn_ballot_w64(bad);
      if (mask != 0) {
        const int tile = (k * kThreads + kWave * wave) / kTile + ((uint32_t)mask == 0u ? 1 : 0);
        first_dirty = tile < first_dirty ? tile : first_dirty;
      }
    }
    if (lane == 0) sm.first_dirty[wave] = first_dirty;
    __syncthreads();
  }
  int first_dirty;
  if (arith || page_arith) {
    // tile t is clean when its keys all lie inside the split and at or before minpos
    const int c1 = minpos - e_begin - (kTile - 1);
    const int fd1 = c1 < 0 ? 0 : c1 / kTile + 1;
    const int fd2 = (e_end - e_begin) / kTile;
    first_dirty = fd1 < fd2 ? fd1 : fd2;
    if (page_bad) first_dirty = 0;
  } else {
    first_dirty = sm.first_dirty[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) first_dirty = sm.first_dirty[w] < first_dirty ? sm.first_dirty[w] : first_dirty;
    first_dirty = __builtin_amdgcn_readfirstlane(first_dirty);
  }
  const bool want_lx = (gather ? p.lse_g : p.lse_f) != nullptr;

  RowState<NT> st;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    st.m[nt] = -INFINITY;
    st.l[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    st.lx[nt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) st.o[nt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // ---- stream this wave's tiles (tile w, w+4, ...) through its two LDS slots.  The waits are
  // explicit: the tile about to be read was issued kTileLoads loads before the newest ones.
  if (wave < ntiles) {
    uint8_t* slot_a = sm.u.slots.ring[wave][0];
    uint8_t* slot_b = sm.u.slots.ring[wave][1];
    const uint32_t slot_a_lds = lds_addr(slot_a), slot_b_lds = lds_addr(slot_b);
    TileRows A;
    TileRegs<NT, PAGED> T;
    if (arith) {
      // row offset (16-byte units) of key e_begin + slot: one scalar term per tile, lane-constant rest;
      // keys of the ragged last tile past the split stay in the allocation through the clamp in
      // dma_tile and are masked by their positions
      const uint32_t base16 = (uint32_t)(((int64_t)s * p.kv.stride_seq + (int64_t)g * p.kv.stride_head) >> 3);
      const uint32_t tok16 = (uint32_t)(p.kv.stride_tok >> 3);
      const uint32_t off_k0 = (uint32_t)lr * tok16, off_k1 = (uint32_t)(16 + lr) * tok16;
      const uint32_t off_v = (uint32_t)(4 * lg) * tok16;
      auto rows_at = [&](int slot0) {
        if (slot0 >= ntiles * kTile) {   // a padding tile past this wave's last: row 0, a cache-resident address
          A.k[0] = A.k[1] = 0u;
#pragma unroll
          for (int h = 0; h < 2; ++h) A.v[h] = u32x4{0u, 0u, 0u, 0u};
          return;
        }
        const uint32_t r0 = base16 + (uint32_t)(e_begin + slot0) * tok16;
        A.k[0] = r0 + off_k0;
        A.k[1] = r0 + off_k1;
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int i = 0; i < 4; ++i) A.v[h][i] = r0 + (uint32_t)(16 * h + i) * tok16 + off_v;
      };
      auto pos_at = [&](int slot0) {
        return [=](int i) {
          const int e = e_begin + slot0 + 16 * (i >> 2) + 4 * lg + (i & 3);
          return e < e_end ? e : -1;
        };
      };
      rows_at(kTile * wave);
      dma_tile(p.kv, A, p.max_roff, slot_a, lane, !gather);
      rows_at(kTile * (wave + kWaves));
      dma_tile(p.kv, A, p.max_roff, slot_b, lane, !gather);
      for (int it = wave;; it += 2 * kWaves) {
        asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
        read_tile<NT, PAGED>(T, slot_a_lds, lane);
        rows_at(kTile * (it + 2 * kWaves));
        dma_tile(p.kv, A, p.max_roff, slot_a, lane, !gather);
        tile_step<NT, PAGED>(st, T, qop, rowpos, p.scale_log2, it >= first_dirty, want_lx, pos_at(kTile * it), pass_v(T));
        if (it + kWaves >= ntiles) break;
        asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
        read_tile<NT, PAGED>(T, slot_b_lds, lane);
        rows_at(kTile * (it + 3 * kWaves));
        dma_tile(p.kv, A, p.max_roff, slot_b, lane, !gather);
        tile_step<NT, PAGED>(st, T, qop, rowpos, p.scale_log2, it + kWaves >= first_dirty, want_lx,
                             pos_at(kTile * (it + kWaves)), pass_v(T));
        if (it + 2 * kWaves >= ntiles) break;
      }
    } else if (page_arith) {
      // row offset of key t = offset of its page (LDS table) + (t % page_size) * stride_tok.  A tile
      // starts at a multiple of 32 keys, so each 16-key sub-tile lies in one page; vb bit h records
      // whether sub-tile h's page is in the pool (absent keys are masked by their positions)
      const uint32_t roff_lds = lds_addr(sm.u.slots.roff);
      const uint32_t tok16 = (uint32_t)(p.kv.stride_tok >> 3);
      const int P = p.kv.page_size;
      const uint32_t off_k = (uint32_t)lr, off_v = (uint32_t)(4 * lg);
      auto rows_at = [&](int slot0, uint32_t& vb) {
        vb = 0u;
        if (slot0 >= ntiles * kTile) {   // a padding tile past this wave's last: row 0, a cache-resident address
          A.k[0] = A.k[1] = 0u;
#pragma unroll
          for (int h = 0; h < 2; ++h) A.v[h] = u32x4{0u, 0u, 0u, 0u};
          return;
        }
        uint32_t a[2], w[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int t = e_begin + slot0 + 16 * h;
          const int pi = div_small(t >> 4, psub, inv_psub);
          // a sub-tile wholly past the split reads entry 0 (always loaded) and is masked anyway
          const int j = t < e_end ? pi - page0 : 0;
          a[h] = roff_lds + 4 * (uint32_t)j;
          w[h] = (uint32_t)(t - pi * P);
        }
        uint32_t b[2];
        asm volatile(
            "ds_read_b32 %0, %2\n"
            "ds_read_b32 %1, %3\n"
            "s_waitcnt lgkmcnt(0)"
            : "=&v"(b[0]), "=&v"(b[1])
            : "v"(a[0]), "v"(a[1]));
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const bool ok = b[h] != 0xFFFFFFFFu;
          vb |= ok ? (1u << h) : 0u;
          const uint32_t base = ok ? b[h] : 0u;
          A.k[h] = base + (w[h] + off_k) * tok16;
#pragma unroll
          for (int i = 0; i < 4; ++i) A.v[h][i] = base + (w[h] + off_v + (uint32_t)i) * tok16;
        }
      };
      auto pos_at = [&](int slot0, uint32_t vb) {
        return [=](int i) {
          const int e = e_begin + slot0 + 16 * (i >> 2) + 4 * lg + (i & 3);
          return (e < e_end && ((vb >> (i >> 2)) & 1u)) ? e : -1;
        };
      };
      uint32_t vb_a, vb_b;
      rows_at(kTile * wave, vb_a);
      dma_tile(p.kv, A, p.max_roff, slot_a, lane, true);
      rows_at(kTile * (wave + kWaves), vb_b);
      dma_tile(p.kv, A, p.max_roff, slot_b, lane, true);
      for (int it = wave;; it += 2 * kWaves) {
        asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
        read_tile<NT, PAGED>(T, slot_a_lds, lane);
        const uint32_t vb_now = vb_a;
        rows_at(kTile * (it + 2 * kWaves), vb_a);
        dma_tile(p.kv, A, p.max_roff, slot_a, lane, true);
        tile_step<NT, PAGED>(st, T, qop, rowpos, p.scale_log2, it >= first_dirty, want_lx, pos_at(kTile * it, vb_now),
                             pass_v(T));
        if (it + kWaves >= ntiles) break;
        asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
        read_tile<NT, PAGED>(T, slot_b_lds, lane);
        const uint32_t vb_next = vb_b;
        rows_at(kTile * (it + 3 * kWaves), vb_b);
        dma_tile(p.kv, A, p.max_roff, slot_b, lane, true);
        tile_step<NT, PAGED>(st, T, qop, rowpos, p.scale_log2, it + kWaves >= first_dirty, want_lx,
                             pos_at(kTile * (it + kWaves), vb_next), pass_v(T));
        if (it + 2 * kWaves >= ntiles) break;
      }
    } else {
      const uint32_t roff_lds = lds_addr(sm.u.slots.roff);
      const uint32_t tpos_lds = lds_addr(sm.u.slots.tpos);
      auto pos_of = [&](int i) { return (int)T.tp[i >> 2][i & 3]; };
      read_rows(A, roff_lds, kTile * wave, lane);
      dma_tile(p.kv, A, p.max_roff, slot_a, lane, !gather);
      read_rows(A, roff_lds, kTile * (wave + kWaves), lane);
      dma_tile(p.kv, A, p.max_roff, slot_b, lane, !gather);
      for (int it = wave;; it += 2 * kWaves) {
        asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
        read_tile_and_rows<NT, PAGED>(T, A, slot_a_lds, tpos_lds, kTile * it, roff_lds, kTile * (it + 2 * kWaves),
                                      lane);
        dma_tile(p.kv, A, p.max_roff, slot_a, lane, !gather);
        tile_step<NT, PAGED>(st, T, qop, rowpos, p.scale_log2, it >= first_dirty, want_lx, pos_of, pass_v(T));
        if (it + kWaves >= ntiles) break;
        asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
        read_tile_and_rows<NT, PAGED>(T, A, slot_b_lds, tpos_lds, kTile * (it + kWaves), roff_lds,
                                      kTile * (it + 3 * kWaves), lane);
        dma_tile(p.kv, A, p.max_roff, slot_b, lane, !gather);
        tile_step<NT, PAGED>(st, T, qop, rowpos, p.scale_log2, it + kWaves >= first_dirty, want_lx, pos_of, pass_v(T));
        if (it + 2 * kWaves >= ntiles) break;
      }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // padding loads land before the LDS is reused
  }
  __syncthreads();   // the slot table is dead from here on; its LDS becomes the merge buffer

  // ---- wave state -> LDS: row r = 16*nt + lane%16; lane group lg holds d in [32lg, 32lg+32)
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const float l = st.l[nt][0];
    float lx = st.lx[nt];
    lx += shfl_xor_f(lx, 16);
    lx += shfl_xor_f(lx, 32);
    const int r = 16 * nt + lr;
    if (lg == 0) {
      sm.u.merge.m[wave][r] = st.m[nt];
      sm.u.merge.l[wave][r] = l;
      sm.u.merge.lx[wave][r] = lx;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float* dst = &sm.u.merge.o[wave][r][32 * lg + 8 * i];
      *reinterpret_cast<f32x4*>(dst) = f32x4{st.o[nt][0][i], st.o[nt][1][i], st.o[nt][2][i], st.o[nt][3][i]};
      *reinterpret_cast<f32x4*>(dst + 4) = f32x4{st.o[nt][4][i], st.o[nt][5][i], st.o[nt][6][i], st.o[nt][7][i]};
    }
  }
  __syncthreads();

  // ---- merge the 4 waves: thread -> (row, d range)
  constexpr int kPerThread = RB::kRows * kD / kThreads;   // 8 (NT=1) or 16 (NT=2)
  const int r = tid / (kD / kPerThread);
  const int d0 = (tid % (kD / kPerThread)) * kPerThread;
  float M = -INFINITY;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) M = fmaxf(M, sm.u.merge.m[w][r]);
  const float Muse = M == -INFINITY ? 0.f : M;
  float Lsum = 0.f, Lx = 0.f, acc[kPerThread];
#pragma unroll
  for (int e = 0; e < kPerThread; ++e) acc[e] = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const float wt = exp2f(sm.u.merge.m[w][r] - Muse);
    Lsum += wt * sm.u.merge.l[w][r];
    Lx += wt * sm.u.merge.lx[w][r];
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) acc[e] += wt * sm.u.merge.o[w][r][d0 + e];
  }

  const int n = rb * RB::kRows + r;
  const bool row_valid = n < p.R;
  const int jrow = row_valid ? n / p.G : 0;
  const int hrow = g * p.G + (row_valid ? n % p.G : 0);
  const int64_t orow = ((int64_t)s * p.nq + jrow) * p.Hq + hrow;     // row within [S][nq][Hq]
  const int64_t view_rows = (int64_t)p.S * p.nq * p.Hq;
  uint16_t* out = gather ? p.out_g + (int64_t)view * view_rows * kD : p.out_f;
  float* lse = gather ? (p.lse_g ? p.lse_g + (int64_t)view * view_rows : nullptr) : p.lse_f;

  auto write_final = [&](float Mf, float Lf, float Lxf, const float* a) {
    if (!row_valid) return;
    const float inv = Lf > 0.f ? 1.f / Lf : 0.f;
    uint32_t w[kPerThread / 2];
#pragma unroll
    for (int e = 0; e < kPerThread; e += 2) w[e / 2] = pack_bf16x2(a[e] * inv, a[e + 1] * inv);
    uint16_t* dst = out + orow * kD + d0;
#pragma unroll
    for (int e = 0; e < kPerThread / 8; ++e)
      *reinterpret_cast<u32x4*>(dst + 8 * e) = u32x4{w[4 * e], w[4 * e + 1], w[4 * e + 2], w[4 * e + 3]};
    if (lse && d0 == 0) lse[orow] = Lxf > 0.f ? (Mf + __log2f(Lxf)) * kLn2 : -INFINITY;
  };

  if (nsplit == 1) {
    write_final(M, Lsum, Lx, acc);
    return;
  }

  // ---- publish this split's partial record (rows that exist only); the last split merges them.
  // Record layout: row stats as one float4 per row, then the outputs thread-major (4-float chunk c
  // of thread t at chunk index c*kThreads + t), so each store instruction of a wave writes 1 KiB
  // contiguously; the merging workgroup reads with the same thread mapping.
  const float* rec_base = p.part + (gather ? 0 : (int64_t)p.units_g * p.nsplit_g * RB::kRec);
  const int unit_local = gather ? unit : unit - p.units_g;
  const __amdgpu_buffer_rsrc_t urec =
      make_rsrc(rec_base + (int64_t)unit_local * nsplit * RB::kRec, (uint32_t)(nsplit * RB::kRec * 4));
  constexpr int kChunks = kPerThread / 4;
  constexpr uint32_t kOutOff = 16 * RB::kRows;
  if constexpr (!TWO_LEVEL) {
    // verify's records (NT = 2) hold the unnormalised outputs in bf16, eight per 16 bytes; the row
    // statistics stay fp32.  A merged output is a weighted mean of the records' rows, so their
    // rounding (relative 2^-9) adds at most 2^-9 of the output's scale before its own bf16 rounding.
    constexpr bool kBf16 = NT == 2;
    constexpr int kWords = kBf16 ? kChunks / 2 : kChunks;     // 16-byte output words per thread
    if (row_valid) {
      const uint32_t rec = (uint32_t)split * RB::kRec * 4;
      if (d0 == 0) store16_coherent(urec, rec + 16 * r, f32x4{M, Lsum, Lx, 0.f});
  #pragma unroll
      for (int c = 0; c < kWords; ++c) {
        const uint32_t off = rec + kOutOff + 16 * (c * kThreads + tid);
        if constexpr (kBf16)
          store16_coherent(urec, off, as_f32x4(pack_record_bf16(f32x4{acc[8 * c], acc[8 * c + 1], acc[8 * c + 2], acc[8 * c + 3]},
                                                                f32x4{acc[8 * c + 4], acc[8 * c + 5], acc[8 * c + 6], acc[8 * c + 7]})));
        else
          store16_coherent(urec, off, f32x4{acc[4 * c], acc[4 * c + 1], acc[4 * c + 2], acc[4 * c + 3]});
      }
    }
    wait_vmem();
    __syncthreads();
    if (tid == 0) sm.last = arrive(counter_line(p.counters, unit), (uint32_t)nsplit);
    __syncthreads();
    if (!sm.last) return;
    if (tid == 0) reset_counter(counter_line(p.counters, unit));   // ready for the next call
    if (!row_valid) return;

    // merge the splits in split order with an online rescale, a batch of records at a time; every
    // load of a batch is issued before any of its results is used
    constexpr int kBatch = 8;
    float Mg = -INFINITY, Lg = 0.f, Lxg = 0.f, ag[kPerThread];
  #pragma unroll
    for (int e = 0; e < kPerThread; ++e) ag[e] = 0.f;
    for (int sp0 = 0; sp0 < nsplit; sp0 += kBatch) {
      f32x4 sv[kBatch], ow[kBatch][kWords];
  #pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const uint32_t rec = (uint32_t)(sp0 + u) * RB::kRec * 4;
        const bool ok = sp0 + u < nsplit;
        sv[u] = ok ? load16_coherent(urec, rec + 16 * r) : f32x4{-INFINITY, 0.f, 0.f, 0.f};
  #pragma unroll
        for (int c = 0; c < kWords; ++c)
          ow[u][c] = ok ? load16_coherent(urec, rec + kOutOff + 16 * (c * kThreads + tid)) : f32x4{0.f, 0.f, 0.f, 0.f};
      }
      float mb = Mg;
  #pragma unroll
      for (int u = 0; u < kBatch; ++u) mb = fmaxf(mb, sv[u][0]);
      const float mbu = mb == -INFINITY ? 0.f : mb;
      const float sc = exp2f(Mg - mbu);
      Lg *= sc;
      Lxg *= sc;
  #pragma unroll
      for (int e = 0; e < kPerThread; ++e) ag[e] *= sc;
  #pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const float wt = exp2f(sv[u][0] - mbu);
        Lg += wt * sv[u][1];
        Lxg += wt * sv[u][2];
        f32x4 ov[kChunks];
        if constexpr (kBf16) {
  #pragma unroll
          for (int c = 0; c < kWords; ++c) unpack_record_bf16(as_u32x4(ow[u][c]), ov[2 * c], ov[2 * c + 1]);
        } else {
  #pragma unroll
          for (int c = 0; c < kChunks; ++c) ov[c] = ow[u][c];
        }
  #pragma unroll
        for (int c = 0; c < kChunks; ++c)
  #pragma unroll
          for (int i = 0; i < 4; ++i) ag[4 * c + i] += wt * ov[c][i];
      }
      Mg = mb;
    }
    write_final(Mg, Lg, Lxg, ag);
  } else {
    auto store_record = [&](int slot, float Mr, float Lr, float Lxr, const float* a) {
      if (!row_valid) return;
      const uint32_t rec = (uint32_t)slot * RB::kRec * 4;
      if (d0 == 0) store16_coherent(urec, rec + 16 * r, f32x4{Mr, Lr, Lxr, 0.f});
  #pragma unroll
      for (int c = 0; c < kChunks; ++c)
        store16_coherent(urec, rec + kOutOff + 16 * (c * kThreads + tid),
                         f32x4{a[4 * c], a[4 * c + 1], a[4 * c + 2], a[4 * c + 3]});
    };
    // Merge `count` records at slots first, first + stride, ... in that order with an online rescale,
    // a batch of records at a time (every load of a batch issued before any of its results is used).
    float Mg, Lg, Lxg, ag[kPerThread];
    auto merge_records = [&](int first, int count, int stride) {
      Mg = -INFINITY;
      Lg = Lxg = 0.f;
  #pragma unroll
      for (int e = 0; e < kPerThread; ++e) ag[e] = 0.f;
      if (!row_valid) return;
      for (int sp0 = 0; sp0 < count; sp0 += kMergeGroup) {
        f32x4 sv[kMergeGroup], ov[kMergeGroup][kChunks];
  #pragma unroll
        for (int u = 0; u < kMergeGroup; ++u) {
          const uint32_t rec = (uint32_t)(first + (sp0 + u) * stride) * RB::kRec * 4;
          const bool ok = sp0 + u < count;
          sv[u] = ok ? load16_coherent(urec, rec + 16 * r) : f32x4{-INFINITY, 0.f, 0.f, 0.f};
  #pragma unroll
          for (int c = 0; c < kChunks; ++c)
            ov[u][c] = ok ? load16_coherent(urec, rec + kOutOff + 16 * (c * kThreads + tid))
                          : f32x4{0.f, 0.f, 0.f, 0.f};
        }
        float mb = Mg;
  #pragma unroll
        for (int u = 0; u < kMergeGroup; ++u) mb = fmaxf(mb, sv[u][0]);
        const float mbu = mb == -INFINITY ? 0.f : mb;
        const float sc = exp2f(Mg - mbu);
        Lg *= sc;
        Lxg *= sc;
  #pragma unroll
        for (int e = 0; e < kPerThread; ++e) ag[e] *= sc;
  #pragma unroll
        for (int u = 0; u < kMergeGroup; ++u) {
          const float wt = exp2f(sv[u][0] - mbu);
          Lg += wt * sv[u][1];
          Lxg += wt * sv[u][2];
  #pragma unroll
          for (int c = 0; c < kChunks; ++c)
  #pragma unroll
            for (int i = 0; i < 4; ++i) ag[4 * c + i] += wt * ov[u][c][i];
        }
        Mg = mb;
      }
    };

    // A unit of at most kMergeGroup splits is merged by its last split.  A larger one merges in two
    // levels, each one batch of loads: the last split of each group of kMergeGroup consecutive splits
    // merges the group into the group's first slot, and the last group merges the groups in order.
    store_record(split, M, Lsum, Lx, acc);
    const bool two_level = nsplit > kMergeGroup;
    const int grp = split / kMergeGroup;
    const int ngroups = (nsplit + kMergeGroup - 1) / kMergeGroup;
    const int g_first = two_level ? grp * kMergeGroup : 0;
    const int g_count = two_level ? (nsplit - g_first < kMergeGroup ? nsplit - g_first : kMergeGroup) : nsplit;
    wait_vmem();
    __syncthreads();
    if (tid == 0) {
      uint32_t* c = two_level ? counter_line(p.counters, p.units_all + (int64_t)unit * p.ngrp + grp)
                              : counter_line(p.counters, unit);
      const bool last = arrive(c, (uint32_t)g_count);
      if (last) reset_counter(c);                      // ready for the next call
      sm.last = last;
    }
    __syncthreads();
    if (!sm.last) return;
    merge_records(g_first, g_count, 1);
    if (!two_level) {
      write_final(Mg, Lg, Lxg, ag);
      return;
    }
    __syncthreads();   // every row's loads of the group's first slot are done before it is rewritten
    store_record(g_first, Mg, Lg, Lxg, ag);
    wait_vmem();
    __syncthreads();
    if (tid == 0) {
      uint32_t* c = counter_line(p.counters, unit);
      const bool last = arrive(c, (uint32_t)ngroups);
      if (last) reset_counter(c);
      sm.last = last;
    }
    __syncthreads();
    if (!sm.last) return;
    merge_records(0, ngroups, kMergeGroup);
    write_final(Mg, Lg, Lxg, ag);
  }
}

// ---- block mode: many query rows per (sequence, KV head) ---------------------
//
// When a unit has more than one 32-row block (the multiview continuation block:
// C x G rows), re-streaming K/V once per row block would multiply the traffic.
// A block-mode workgroup has 8 waves, wave w owning row block 8*rg + w, and all
// of them consume every 32-key tile of its range from a shared LDS ring: each
// wave issues 2 of a tile's 16 direct-to-LDS loads, and one barrier per two
// tiles both publishes the next two landed tiles and frees the two slots read
// before it.  The ranges are equal shares of the (sequence, KV head, row
// group)'s whole key stream, every view and the full branch in turn, cut at run
// time when the views' lengths are known; pieces of a branch met by several
// workgroups leave per-row-block records that block_merge_kernel combines.

constexpr int kBWaves = 8;
constexpr int kBThreads = kBWaves * kWave;
constexpr int kBRing = 7;                          // tile slots: the two being read, up to five in flight
constexpr int kBMaxPieces = 64;                    // branches per unit (host-checked)
// a workgroup's range holds at most kMaxSplitKeys entries, each piece pads its last tile, and the
// prefetches run kBRing tiles past the end
constexpr int kBSlotCap = kMaxSplitKeys + (kBMaxPieces + kBRing) * kTile;
// a block-mode tile: K in the score operand order (8 KiB), then V row-major for the transposing reads
constexpr int kBTileBytes = 8192 + kRmTileBytes;

// One piece of a workgroup's range: entries [e0, e1) of branch b, from slot-table tile t0; the
// branch spans nwg workgroups, its records start at slot `slot`, this piece's is number wo.
struct BlockPiece {
  int32_t b, e0, e1, t0, nwg, slot, wo;
};
// A piece read from LDS, made wave-uniform: the record address built from it then stays in scalar
// registers (a per-lane address would turn every record store into a loop over distinct values).
__device__ inline BlockPiece uniform_piece(const BlockPiece& x) {
  return BlockPiece{__builtin_amdgcn_readfirstlane(x.b), __builtin_amdgcn_readfirstlane(x.e0),
                    __builtin_amdgcn_readfirstlane(x.e1), __builtin_amdgcn_readfirstlane(x.t0),
                    __builtin_amdgcn_readfirstlane(x.nwg), __builtin_amdgcn_readfirstlane(x.slot),
                    __builtin_amdgcn_readfirstlane(x.wo)};
}

struct BlockSmem {
  alignas(16) int32_t roff[kBSlotCap];
  alignas(16) int32_t tpos[kBSlotCap];
  alignas(16) uint8_t ring[kBRing][kBTileBytes];
  BlockPiece pc[kBMaxPieces];
  int32_t blen[kBMaxPieces];                       // branch lengths
};

// Load q (0..15) of a tile for this lane; `r` is the row's offset in 16-byte units.  K loads
// q < 8 (sub-tile q/4, k-step q%4) land in the score operand order.  V loads q >= 8 fill the
// tile's second half as a row-major tile for the transposing reads (rm_row, rm_chunk).
__device__ inline void dma_load(const KvView& kv, uint32_t r, uint32_t max_roff, int q, uint8_t* dst, int lane) {
  const int lg = lane >> 4, lr = lane & 15;
  const uint32_t ro = r < max_roff ? r : max_roff;
  if (q < 8) dma16(kv.k + ((uint64_t)ro << 3) + 32 * lg + 8 * (q & 3), dst + q * 1024);
  else dma16(kv.v + ((uint64_t)ro << 3) + 8 * rm_chunk(lane), dst + 8192 + rm_block_off(q - 8));
}

// ---- block mode's tile step, split for software pipelining -------------------
//
// Step t of a wave computes the scores of tile t+1 on the matrix cores while the vector units turn
// the scores of tile t into weights (phase A), then the PV product of tile t while the vector units
// take the row maxima of tile t+1 (phase B).  Neither half's MFMA work depends on its VALU work, so
// one wave keeps both units busy instead of alternating between them.  Per tile the arithmetic is
// the split kernel's tile_step (plus the two-term weights of the training outputs), in the same
// order, with the V^T operands from transposing LDS reads.

// Scores S^T = K Q^T of one tile (unscaled): sub-tile sub, register r of lane l holds key
// 16*sub + 4*(l/16) + r of row 16*nt + l%16.
template <int NT>
__device__ inline void block_qk(f32x4 (&s)[2][NT], const u32x4 (&k)[2][4], const bf16x8 (&qop)[NT][4]) {
  const f32x4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        s[sub][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(k[sub][j]), qop[nt][j], j == 0 ? z : s[sub][nt],
                                                             0, 0, 0);
}

// Scores of absent keys and of keys past a row's position -> -inf.
template <int NT>
__device__ inline void block_mask(f32x4 (&s)[2][NT], const u32x4 (&tp)[2], const int (&rowpos)[NT]) {
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int tpos = (int)tp[i >> 2][i & 3];
      if (!(tpos >= 0 && tpos <= rowpos[nt])) s[i >> 2][nt][i & 3] = -INFINITY;
    }
}

// Row maxima of a tile's scaled scores (log2 domain), shared by the row's 4 lane groups.
template <int NT>
__device__ inline void block_tile_max(float (&mx)[NT], const f32x4 (&s)[2][NT], float scale_log2) {
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float v = -INFINITY;
#pragma unroll
    for (int i = 0; i < 8; ++i) v = fmaxf(v, s[i >> 2][nt][i & 3]);
    mx[nt] = max_xor32(max_xor16(v)) * scale_log2;    // scale > 0: the max commutes with it
  }
}

// Raise the reference max of rows whose tile max exceeds it by more than kSlack, rescaling their
// accumulators (the lazy rescale of tile_step).
template <int NT>
__device__ inline void block_raise(RowState<NT>& st, const float (&mx)[NT]) {
  bool raise = false;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) raise |= mx[nt] > st.m[nt] + kSlack;
  if (__builtin_expect(__builtin_amdgcn_ballot_w64(raise) != 0, 0)) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const bool up = mx[nt] > st.m[nt] + kSlack;
      const float alpha = up ? __builtin_amdgcn_exp2f(st.m[nt] - mx[nt]) : 1.f;   // 0 on the first visible tile
      st.m[nt] = up ? mx[nt] : st.m[nt];
      st.l[nt] *= alpha;
      st.lx[nt] *= alpha;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) st.o[nt][dt] *= alpha;
    }
  }
}

// Weights of a tile against the reference max, rounded to bf16 for the PV product, summed into the
// normaliser by MFMA (which then sums exactly the rounded weights the PV product sees); `w` keeps
// them unrounded for the log-sum-exp sum.  TRAIN: each weight enters the PV product and the
// normaliser as a bf16 pair hi + lo (lo the rounded remainder), so the output carries the weights to
// about 2^-17 instead of 2^-9: the fp32 output then serves the backward's <dO, O> (which cancels
// against <dO, v_t>) without amplifying rounding.
template <int NT, bool TRAIN>
__device__ inline void block_weights(RowState<NT>& st, const f32x4 (&s)[2][NT], float scale_log2, bf16x8 (&pop)[NT],
                                     bf16x8 (&plo)[NT], float (&w)[NT][8]) {
  const bf16x8 ones = as_bf16x8(u32x4{0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u});
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const float muse = st.m[nt] == -INFINITY ? 0.f : st.m[nt];
#pragma unroll
    for (int i = 0; i < 8; ++i) w[nt][i] = __builtin_amdgcn_exp2f(fmaf(s[i >> 2][nt][i & 3], scale_log2, -muse));
    u32x4 pw;
#pragma unroll
    for (int i = 0; i < 4; ++i) pw[i] = pack_bf16x2(w[nt][2 * i], w[nt][2 * i + 1]);
    pop[nt] = as_bf16x8(pw);
    if constexpr (TRAIN) {
      u32x4 lw;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        lw[i] = pack_bf16x2(w[nt][2 * i] - bf16_lo(pw[i]), w[nt][2 * i + 1] - bf16_hi(pw[i]));
      plo[nt] = as_bf16x8(lw);
      st.l[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, plo[nt], st.l[nt], 0, 0, 0);
    }
    st.l[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pop[nt], st.l[nt], 0, 0, 0);
  }
}

template <int NT, bool TRAIN>
__device__ inline void block_pv(RowState<NT>& st, const bf16x8 (&vt)[8], const bf16x8 (&pop)[NT],
                                const bf16x8 (&plo)[NT]) {
#pragma unroll
  for (int dt = 0; dt < 8; ++dt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      st.o[nt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vt[dt], pop[nt], st.o[nt][dt], 0, 0, 0);
      if constexpr (TRAIN) st.o[nt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vt[dt], plo[nt], st.o[nt][dt], 0, 0, 0);
    }
}

// Scheduling of a phase: N MFMAs, each followed by up to V vector instructions (transcendentals
// included), so that the in-order issue of one wave alternates between the two units.
template <int N, int V>
__device__ inline void interleave_mfma_valu() {
#pragma unroll
  for (int i = 0; i < N; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x402, V, 0);
  }
}

// K and the key positions of the tile in LDS slot `slot` (lane's part at slot + 16*lane), one
// statement ending in its own wait.
__device__ inline void read_block_k(u32x4 (&k)[2][4], u32x4 (&tp)[2], uint32_t slot, uint32_t ap, int lane) {
  const uint32_t at = slot + 16 * lane;
  asm volatile(
      "ds_read_b128 %0, %10\n"
      "ds_read_b128 %1, %10 offset:1024\n"
      "ds_read_b128 %2, %10 offset:2048\n"
      "ds_read_b128 %3, %10 offset:3072\n"
      "ds_read_b128 %4, %10 offset:4096\n"
      "ds_read_b128 %5, %10 offset:5120\n"
      "ds_read_b128 %6, %10 offset:6144\n"
      "ds_read_b128 %7, %10 offset:7168\n"
      "ds_read_b128 %8, %11\n"
      "ds_read_b128 %9, %11 offset:64\n"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(k[0][0]), "=&v"(k[0][1]), "=&v"(k[0][2]), "=&v"(k[0][3]), "=&v"(k[1][0]), "=&v"(k[1][1]),
        "=&v"(k[1][2]), "=&v"(k[1][3]), "=&v"(tp[0]), "=&v"(tp[1])
      : "v"(at), "v"(ap));
}

// The transposing V reads of read_vt_tr split in two: issue_vt_tr starts them without waiting, so they
// run under the MFMA and VALU work that follows; wait_vt_tr waits for them and unpacks the operands.
// The raw registers pass from one statement to the other as in-out operands, so nothing reads them
// before the wait.
__device__ inline void issue_vt_tr(uint64_t (&x)[16], uint32_t slot, const uint32_t (&vo)[4]) {
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
      "ds_read_b64_tr_b16 %15, %19 offset:4136"
      : "=&v"(x[0]), "=&v"(x[1]), "=&v"(x[2]), "=&v"(x[3]), "=&v"(x[4]), "=&v"(x[5]), "=&v"(x[6]), "=&v"(x[7]),
        "=&v"(x[8]), "=&v"(x[9]), "=&v"(x[10]), "=&v"(x[11]), "=&v"(x[12]), "=&v"(x[13]), "=&v"(x[14]),
        "=&v"(x[15])
      : "v"(slot + vo[0]), "v"(slot + vo[1]), "v"(slot + vo[2]), "v"(slot + vo[3]));
}
__device__ inline void wait_vt_tr(bf16x8 (&vt)[8], uint64_t (&x)[16]) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(x[0]), "+v"(x[1]), "+v"(x[2]), "+v"(x[3]), "+v"(x[4]), "+v"(x[5]), "+v"(x[6]), "+v"(x[7]),
                 "+v"(x[8]), "+v"(x[9]), "+v"(x[10]), "+v"(x[11]), "+v"(x[12]), "+v"(x[13]), "+v"(x[14]),
                 "+v"(x[15]));
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) {
    const uint64_t lo = x[2 * dt], hi = x[2 * dt + 1];
    vt[dt] = as_bf16x8(u32x4{(uint32_t)lo, (uint32_t)(lo >> 32), (uint32_t)hi, (uint32_t)(hi >> 32)});
  }
}

// Whether a tile needs the visibility mask for a wave whose earliest row sits at `minpos`: some slot
// absent (-1) or past minpos.  As unsigned, -1 exceeds every position.
__device__ inline bool block_dirty(const u32x4 (&tp)[2], int minpos) {
  const uint32_t a = max(max(tp[0][0], tp[0][1]), max(tp[0][2], tp[0][3]));
  const uint32_t b = max(max(tp[1][0], tp[1][1]), max(tp[1][2], tp[1][3]));
  const bool bad = minpos < 0 || max(a, b) > (uint32_t)minpos;
  return __builtin_amdgcn_ballot_w64(bad) != 0;
}

// Split records of the bf16-output path keep the unnormalised outputs in bf16: two d-tiles of one
// lane in 16 bytes.  Each merged output is a weighted mean of the records' rows, so their rounding
// (relative 2^-9 per element) adds at most 2^-9 of the output's scale before its own bf16 rounding.
// The training path (fp32 outputs) keeps fp32 records.
// Workgroup barrier for LDS traffic: waits for this wave's LDS operations only, not for its global
// loads in flight.
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Branch b's outputs of row block rb (rows 16*nt + lane%16 of it) from an unnormalised state:
// register r of d-tile dt holds d = 32*(lane/16) + 4*dt + r.  Rows past R are not written.
template <bool TRAIN>
__device__ inline void block_write_rows(const AttnParams& p, int s, int g, int rb, int b, const float (&M)[2],
                                        const float (&Lw)[2], const float (&Lx)[2], const f32x4 (&o)[2][8],
                                        int lane) {
  constexpr int NT = 2;
  const int lg = lane >> 4, lr = lane & 15;
  const int64_t view_rows = (int64_t)p.S * p.nq * p.Hq;
  const bool gb = b < p.V;
  uint16_t* out = gb ? p.out_g + (int64_t)b * view_rows * kD : p.out_f;
  float* lse = gb ? (p.lse_g ? p.lse_g + (int64_t)b * view_rows : nullptr) : p.lse_f;
  float* out32 = gb ? (p.o32_g ? p.o32_g + (int64_t)b * view_rows * kD : nullptr) : p.o32_f;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int n = rb * RowBlock<NT>::kRows + 16 * nt + lr;
    if (n >= p.R) continue;
    const int j = n / p.G, h = g * p.G + n % p.G;
    const int64_t orow = ((int64_t)s * p.nq + j) * p.Hq + h;
    const float inv = Lw[nt] > 0.f ? 1.f / Lw[nt] : 0.f;
#pragma unroll
    for (int k = 0; k < 4; ++k) {      // d = 32*lg + 8*k + 0..7: d-tiles 2k and 2k+1
      const f32x4 a = o[nt][2 * k] * inv, c = o[nt][2 * k + 1] * inv;
      const u32x4 wv = {pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3]), pack_bf16x2(c[0], c[1]),
                        pack_bf16x2(c[2], c[3])};
      *reinterpret_cast<u32x4*>(out + orow * kD + 32 * lg + 8 * k) = wv;
      if (TRAIN && out32) {
        float* o32 = out32 + orow * kD + 32 * lg + 8 * k;
        *reinterpret_cast<f32x4*>(o32) = a;
        *reinterpret_cast<f32x4*>(o32 + 4) = c;
      }
    }
    if (lse && lg == 0) lse[orow] = Lx[nt] > 0.f ? (M[nt] + __log2f(Lx[nt])) * kLn2 : -INFINITY;
  }
}

// Length of branch b of sequence s in the unit's key stream (the views' entry lists, then the full
// branch's L cache rows).
__device__ inline int block_branch_len(const AttnParams& p, int s, int L, int b) {
  if (b < p.V) {
    const int n = p.nsel[b * p.S + s];
    return n < 0 ? 0 : (n > p.ld_idx ? p.ld_idx : n);
  }
  return L;
}

// Block mode's cut of a unit's key stream (StreamCut): measured, a tile of gathered rows takes
// 1.78 us of a workgroup's loop and a contiguous one 1.43 us.
constexpr int kWGather = 5, kWFull = 4;
using BlockCut = StreamCut<kWGather, kWFull>;

template <bool PAGED, bool TRAIN>
__global__ __launch_bounds__(kBThreads) void block_kernel(AttnParams p) {
  constexpr int NT = 2;
  using RB = RowBlock<NT>;
  __shared__ BlockSmem sm;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lg = lane >> 4, lr = lane & 15;

  // ---- unit (sequence, KV head, row group) and this workgroup's share w of the unit's key stream
  const int bid = xcd_remap(blockIdx.x + fetch_args<false>(p), gridDim.x);   // kernel arguments in one round trip
  const int w = bid % p.nW;
  const int unit = bid / p.nW;
  const int rg = unit % p.n_rg;
  const int pair = unit / p.n_rg;
  const int g = pair % p.Hkv, s = pair / p.Hkv;
  const int rb = rg * kBWaves + wave;            // this wave's row block
  const bool has_rows = rb < p.n_rb;
  const int L = seq_len(p.kv, s);

  // The key stream of a unit is the views' entry lists followed by the full branch's cache rows;
  // its length is known only here (nsel lives on the device), so the unit's nW workgroups cut it
  // into equal ranges at run time.  A range holds one piece per branch it meets, and all its pieces
  // stream through one slot table and one ring.  A branch met by one workgroup is finished there;
  // otherwise each piece leaves a record and the last of the branch's workgroups merges them in
  // stream order.
  // The branch lengths, then the query rows: the rows are needed only at the first tile, so the
  // barriers of the prologue wait for LDS traffic alone (a __syncthreads fence would wait for
  // every global load in flight, the rows' included, at each of them).
  const int blen_t = tid < p.nbr ? block_branch_len(p, s, L, tid) : 0;   // nbr <= kBMaxPieces <= kBThreads

  // ---- query rows of this wave's lanes: row n = rb*32 + 16*nt + lane%16
  bf16x8 qop[NT][4];
  int rowpos[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int n = rb * RB::kRows + 16 * nt + lr;
    const bool valid = n < p.R;
    const int j = valid ? n / p.G : 0;
    const int h = g * p.G + (valid ? n % p.G : 0);
    rowpos[nt] = valid ? L - p.nq + j : 0x7FFFFFFF;
    const uint16_t* qrow = p.q + (((int64_t)s * p.nq + j) * p.Hq + h) * kD + 32 * lg;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) qop[nt][kk] = as_bf16x8(valid ? load16(qrow + 8 * kk) : u32x4{0u, 0u, 0u, 0u});
  }

  if (tid < p.nbr) sm.blen[tid] = blen_t;
  lds_barrier();
  int total = 0, vt = 0;
  for (int b = 0; b < p.nbr; ++b) {
    total += sm.blen[b];
    if (b < p.V) vt += sm.blen[b];
  }
  const BlockCut cut(vt, total, p.nW);
  const int r0 = cut.start_of(w), r1 = cut.start_of(w + 1);
  const int minpos = L - p.nq + (rb * RB::kRows) / p.G;   // earliest row position of this wave

  // ---- the two loads of every tile that this wave issues, and the tile rows they read
  const int q0 = 2 * wave, q1 = 2 * wave + 1;
  auto row_in_tile = [&](int q) { return q < 8 ? 16 * (q >> 2) + lr : rm_row(q - 8, lane); };
  const int rit0 = row_in_tile(q0), rit1 = row_in_tile(q1);
  // transposing V reads (read_vt_tr) of the row-major V half of a tile
  uint32_t vtr_off[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) vtr_off[j] = 8192u + tr_lane_off(lane, j);
  const uint32_t roff_lds = lds_addr(sm.roff), tpos_lds = lds_addr(sm.tpos);
  const uint32_t ring_lds = lds_addr(sm.ring[0]);
  auto issue = [&](int tile, const uint32_t (&r)[2]) {
    uint8_t* dst = sm.ring[tile % kBRing];
    dma_load(p.kv, r[0], p.max_roff, q0, dst, lane);
    dma_load(p.kv, r[1], p.max_roff, q1, dst, lane);
  };

  auto write_rows = [&](int b, const float (&M)[2], const float (&Lw)[2], const float (&Lx)[2],
                        const f32x4 (&o)[2][8]) { block_write_rows<TRAIN>(p, s, g, rb, b, M, Lw, Lx, o, lane); };

  // ---- records of the unit: piece (b, w) at slot base(b) + w - wlo(b), one record per row block
  const int rec_per_unit = p.nW + p.nbr - 1;
  const float* unit_rec = p.part + (int64_t)unit * rec_per_unit * kBWaves * RB::kRec;
  constexpr uint32_t kOutOff = 16 * RB::kRows;

  // ---- this workgroup's pieces, in stream order: entries [e0, e1) of every branch its range meets.
  // A piece takes whole tiles of the slot table (the last one padded), so that a tile never mixes
  // branches.  Empty branches are written by the workgroup whose range holds their place.
  int npc = 0, ntl = 0;
  {
    int off = 0, rbase = 0;
    for (int b = 0; b < p.nbr; ++b) {
      const int n = sm.blen[b];
      const int off_b = off;
      off += n;
      if (n == 0) {
        int owner = cut.wg_of(off_b);
        if (owner > p.nW - 1) owner = p.nW - 1;
        if (owner == w && has_rows) {
          const float m0[NT] = {-INFINITY, -INFINITY}, z[NT] = {0.f, 0.f};
          f32x4 oz[NT][8];
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) oz[nt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
          write_rows(b, m0, z, z, oz);
        }
        continue;
      }
      const int wlo = cut.wg_of(off_b), whi = cut.wg_of(off_b + n - 1);
      const int slot_b = rbase;
      rbase += whi - wlo + 1;
      const int lo = r0 > off_b ? r0 : off_b, hi = r1 < off_b + n ? r1 : off_b + n;
      if (lo >= hi) continue;
      if (tid == 0) {
        sm.pc[npc] = BlockPiece{b, lo - off_b, hi - off_b, ntl, whi - wlo + 1, slot_b, w - wlo};
      }
      ntl += (hi - lo + kTile - 1) / kTile;
      ++npc;
    }
  }
  lds_barrier();

  // ---- one slot table for every piece: all idx (and page-table) loads issued before any is used
  {
    constexpr int kPer = (kBSlotCap + kBThreads - 1) / kBThreads;
    const int nslots = (ntl + kBRing) * kTile;     // padding tiles past the last for the prefetches
    int tv[kPer];
    int k = 0;                                     // piece of this thread's slot (slots increase with j)
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int i = tid + j * kBThreads;
      const int tile = i / kTile;
      while (k + 1 < npc && sm.pc[k + 1].t0 <= tile) ++k;
      int t = -1;
      if (tile < ntl) {
        const BlockPiece pc = sm.pc[k];
        const int e = pc.e0 + (i - kTile * pc.t0);
        if (e < pc.e1) {
          t = pc.b < p.V ? p.idx[(((int64_t)pc.b * p.S + s) * p.Hkv + g) * p.ld_idx + e] : e;
        }
      }
      tv[j] = t;
    }
    int pg[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      tv[j] = (tv[j] >= 0 && tv[j] < L) ? tv[j] : -1;
      if constexpr (PAGED)
        pg[j] = tv[j] >= 0 ? p.kv.page_table[(int64_t)s * p.kv.max_pages_per_seq + tv[j] / p.kv.page_size] : 0;
    }
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int i = tid + j * kBThreads;
      if (i < nslots && i < kBSlotCap) {
        int t = tv[j];
        int64_t o;
        if constexpr (PAGED) {
          o = (unsigned)pg[j] < (unsigned)p.kv.num_pages
                  ? (int64_t)pg[j] * p.kv.stride_page + (int64_t)g * p.kv.stride_head +
                        (int64_t)(t % p.kv.page_size) * p.kv.stride_tok
                  : -1;
        } else {
          o = (int64_t)s * p.kv.stride_seq + (int64_t)g * p.kv.stride_head + (int64_t)t * p.kv.stride_tok;
        }
        if (t < 0 || o < 0) { t = -1; o = 0; }
        sm.roff[i] = (int)(o >> 3);
        sm.tpos[i] = t;
      }
    }
  }
  lds_barrier();

  // ---- stream every tile of every piece through the ring: tiles 0 .. kBRing-3 first
  for (int t = 0; t < kBRing - 2; ++t) {
    uint32_t r[2];
    asm volatile(
        "ds_read_b32 %0, %2\n"
        "ds_read_b32 %1, %3\n"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(r[0]), "=&v"(r[1])
        : "v"(roff_lds + 4 * (kTile * t + rit0)), "v"(roff_lds + 4 * (kTile * t + rit1)));
    issue(t, r);
  }
  // A head step takes the scores of tile 0; step t then finishes tile t and scores tile t+1 (the
  // pipelined step above), reading tile t+1's K and tile t's V^T.  Barriers come at even steps: the
  // one of step t publishes tiles t+1 and t+2 (this wave's loads of them are older than the two tiles
  // issued after them) and certifies that every wave has finished step t-1, so the slots of tiles t-2
  // and t-1 (last read in steps t-2 and t-1) take tiles t+5 and t+6.
  // At the last tile of a piece the wave finishes the piece: its rows' outputs when the piece is the
  // whole branch, else a record (stored now, counted once every piece is done) and a fresh state.
  // A wave without query rows (the row count is not a multiple of the block) only keeps the ring
  // going, with the same barriers.
  static_assert(kBRing == 7, "the wait counts and the issue distance follow the ring depth");
  auto issue_pair = [&](int t) {   // tiles t+5 and t+6, at even steps after the barrier
    uint32_t r[4];
    asm volatile(
        "ds_read_b32 %0, %4\n"
        "ds_read_b32 %1, %5\n"
        "ds_read_b32 %2, %6\n"
        "ds_read_b32 %3, %7\n"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3])
        : "v"(roff_lds + 4 * (kTile * (t + 5) + rit0)), "v"(roff_lds + 4 * (kTile * (t + 5) + rit1)),
          "v"(roff_lds + 4 * (kTile * (t + 6) + rit0)), "v"(roff_lds + 4 * (kTile * (t + 6) + rit1)));
    const uint32_t r5[2] = {r[0], r[1]}, r6[2] = {r[2], r[3]};
    issue(t + 5, r5);
    issue(t + 6, r6);
  };
  if (has_rows) {
    RowState<NT> st;
    auto reset = [&] {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        st.m[nt] = -INFINITY;
        st.l[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        st.lx[nt] = 0.f;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) st.o[nt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    };
    reset();
    int k = 0;
    BlockPiece pc = uniform_piece(sm.pc[0]);
    int t_end = pc.t0 + (pc.e1 - pc.e0 + kTile - 1) / kTile;
    bool want_lx = (pc.b < p.V ? p.lse_g : p.lse_f) != nullptr;
    u32x4 kr[2][4], tp[2];
    f32x4 sc[2][NT];        // scores of the tile this step finishes
    float mx[NT];
    {
      asm volatile("s_waitcnt vmcnt(8)\n\ts_barrier" ::: "memory");   // tile 0 (tiles 1..4 in flight)
      read_block_k(kr, tp, ring_lds, tpos_lds + 4 * (4 * lg), lane);
      block_qk<NT>(sc, kr, qop);
      if (block_dirty(tp, minpos)) block_mask<NT>(sc, tp, rowpos);
      block_tile_max<NT>(mx, sc, p.scale_log2);
      block_raise<NT>(st, mx);
    }
    for (int t = 0; t < ntl; ++t) {
      if ((t & 1) == 0) {
        asm volatile("s_waitcnt vmcnt(4)\n\ts_barrier" ::: "memory");   // tiles t+1, t+2 (t+3, t+4 in flight)
        issue_pair(t);
      }
      read_block_k(kr, tp, ring_lds + (uint32_t)((t + 1) % kBRing) * kBTileBytes,
                   tpos_lds + 4 * (kTile * (t + 1) + 4 * lg), lane);
      uint64_t xv[16];
      issue_vt_tr(xv, ring_lds + (uint32_t)(t % kBRing) * kBTileBytes, vtr_off);
      const bool dirty = block_dirty(tp, minpos);
      // phase A: scores of tile t+1 | weights of tile t
      f32x4 sn[2][NT];
      bf16x8 pop[NT], plo[NT];
      float w[NT][8];
      // raised issue priority for this half: the two waves of a SIMD drift into opposite halves of
      // the step, one issuing score MFMAs and exponentials while the other runs its PV product
      __builtin_amdgcn_s_setprio(1);
      block_qk<NT>(sn, kr, qop);
      block_weights<NT, TRAIN>(st, sc, p.scale_log2, pop, plo, w);
      interleave_mfma_valu<16, 3>();
      __builtin_amdgcn_s_setprio(0);
      if (want_lx) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          float sx = 0.f;
#pragma unroll
          for (int i = 0; i < 8; ++i) sx += w[nt][i];
          st.lx[nt] += sx;
        }
      }
      if (dirty) block_mask<NT>(sn, tp, rowpos);
      bf16x8 vt[8];
      wait_vt_tr(vt, xv);
      // phase B: PV of tile t | row maxima of tile t+1
      block_pv<NT, TRAIN>(st, vt, pop, plo);
      block_tile_max<NT>(mx, sn, p.scale_log2);
      interleave_mfma_valu<(TRAIN ? 32 : 16), 2>();
#pragma unroll
      for (int sub = 0; sub < 2; ++sub)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) sc[sub][nt] = sn[sub][nt];
      if (t + 1 == t_end) {
        // ---- piece k done: per-row (m, l, lx) of rows 16*nt + lane%16
        float lxw[NT], lw[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          float lx = st.lx[nt];
          lx += shfl_xor_f(lx, 16);
          lx += shfl_xor_f(lx, 32);
          lxw[nt] = lx;
          lw[nt] = st.l[nt][0];
        }
        if (pc.nwg == 1) {
          write_rows(pc.b, st.m, lw, lxw, st.o);
        } else {
          // record pc.wo of the branch's pieces for this row block: row stats as float4
          // (m, l, lx, -) per row, then the outputs as chunk x lane 16-byte pieces: chunk (nt, dt) in
          // fp32 on the training path, chunk (nt, d-tile pair) in bf16 otherwise
          const __amdgpu_buffer_rsrc_t urec = make_rsrc(unit_rec + ((int64_t)pc.slot * kBWaves + wave) * RB::kRec,
                                                        (uint32_t)(pc.nwg * kBWaves * RB::kRec * 4));
          const uint32_t rec = (uint32_t)pc.wo * kBWaves * RB::kRec * 4;
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            if (lg == 0) store16_coherent(urec, rec + 16 * (16 * nt + lr), f32x4{st.m[nt], lw[nt], lxw[nt], 0.f});
            if constexpr (TRAIN) {
#pragma unroll
              for (int dt = 0; dt < 8; ++dt)
                store16_coherent(urec, rec + kOutOff + 16 * ((nt * 8 + dt) * kWave + lane), st.o[nt][dt]);
            } else {
#pragma unroll
              for (int q = 0; q < 4; ++q)
                store16_coherent(urec, rec + kOutOff + 16 * ((nt * 4 + q) * kWave + lane),
                                 as_f32x4(pack_record_bf16(st.o[nt][2 * q], st.o[nt][2 * q + 1])));
            }
          }
        }
        reset();
        if (++k < npc) {
          pc = uniform_piece(sm.pc[k]);
          t_end = pc.t0 + (pc.e1 - pc.e0 + kTile - 1) / kTile;
          want_lx = (pc.b < p.V ? p.lse_g : p.lse_f) != nullptr;
        }
      }
      block_raise<NT>(st, mx);
    }
  } else {
    asm volatile("s_waitcnt vmcnt(8)\n\ts_barrier" ::: "memory");
    for (int t = 0; t < ntl; t += 2) {
      asm volatile("s_waitcnt vmcnt(4)\n\ts_barrier" ::: "memory");
      issue_pair(t);
    }
  }

  // records of split branches are merged by block_merge_kernel, launched next on the stream
}

// Merge of the split branches: one wave per (unit, branch, row block, row tile nt, half dh of the
// d-tiles).  The branch's pieces were stored as records by the workgroups of block_kernel that met
// it; they are combined here in stream order with an online rescale and written out.  A separate
// launch spreads the merge over the whole chip: merged by the workgroup that finished last, a branch
// split over 7 workgroups pulled 7 records of 128 KiB into one CU, ~16 us at one CU's bandwidth.
// Every load a wave needs is issued before any result is used: the branch lengths (lane b holds
// branch b's), then up to kMBatch records at a time.  Four records a batch keep the wave at 86 VGPRs
// (bf16 outputs), so the launch's 5120 waves are resident at once; batches of 8 (132 VGPRs, two
// rounds of waves) took 11.1 us on the multiview workload, batches of 4 9.1 us, of 2 9.5 us.
constexpr int kMBatch = 4;
// The merge's kernel arguments, all requested at entry (as fetch_args does for the other kernels):
// fetched where first used they took four round trips before the first record load.
__device__ inline int fetch_merge_args(const AttnParams& p) {
  int z0, z1;
  asm("s_mov_b32 %0, 0" : "=s"(z0) : "s"(p.kv.seq_lens), "s"(p.kv.max_seq_len), "s"(p.nsel), "s"(p.ld_idx), "s"(p.S),
      "s"(p.V), "s"(p.nbr), "s"(p.nW), "s"(p.n_rg), "s"(p.n_rb), "s"(p.Hkv), "s"(p.part));
  asm("s_mov_b32 %0, 0" : "=s"(z1) : "s"(z0), "s"(p.out_g), "s"(p.out_f), "s"(p.lse_g), "s"(p.lse_f), "s"(p.o32_g),
      "s"(p.o32_f), "s"(p.nq), "s"(p.Hq), "s"(p.G), "s"(p.R));
  return z1;
}

template <bool TRAIN>
__global__ __launch_bounds__(4 * kWave) void block_merge_kernel(AttnParams p) {
  constexpr int NT = 2;
  using RB = RowBlock<NT>;
  const int lane = threadIdx.x & (kWave - 1), lg = lane >> 4, lr = lane & 15;
  // the waves work independently (no barrier): four per workgroup, since 5120 single-wave
  // workgroups cost 4.8 us of dispatch alone on the multiview workload
  int id = 4 * blockIdx.x + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) + fetch_merge_args(p);
  const int dh = id & 1, nt = (id >> 1) & 1;
  id >>= 2;
  const int rbl = id % kBWaves;
  const int ub = id / kBWaves;
  const int b = ub % p.nbr, unit = ub / p.nbr;
  const int rg = unit % p.n_rg, pair = unit / p.n_rg;
  const int g = pair % p.Hkv, s = pair / p.Hkv;
  const int rb = rg * kBWaves + rbl;
  if (rb >= p.n_rb) return;
  // lane b holds branch b's length (nbr <= 64 lanes): the views' entry counts are requested before
  // the cache length is waited for, so both loads share one round trip
  const int n_raw = lane < p.V ? p.nsel[lane * p.S + s] : 0;
  const int L = seq_len(p.kv, s);
  const int my_len = lane < p.V ? (n_raw < 0 ? 0 : (n_raw > p.ld_idx ? p.ld_idx : n_raw)) : (lane < p.nbr ? L : 0);
  // the branch's offset in the stream, its length, the stream total and the branch's record slot
  // (one slot per workgroup that met each earlier non-empty branch)
  int total = 0, vt = 0, off_b = 0, n = 0;
  for (int bb = 0; bb < p.nbr; ++bb) {
    const int nb = __builtin_amdgcn_readlane(my_len, bb);
    if (bb == b) { off_b = total; n = nb; }
    total += nb;
    if (bb < p.V) vt += nb;
  }
  const BlockCut cut(vt, total, p.nW);
  if (n == 0) return;
  const int wlo = cut.wg_of(off_b), whi = cut.wg_of(off_b + n - 1);
  const int nwg = whi - wlo + 1;
  if (nwg == 1) return;                            // finished by its one workgroup
  int rbase = 0;
  for (int bb = 0, off = 0; bb < b; ++bb) {
    const int nb = __builtin_amdgcn_readlane(my_len, bb);
    if (nb > 0) rbase += cut.wg_of(off + nb - 1) - cut.wg_of(off) + 1;
    off += nb;
  }
  const int rec_per_unit = p.nW + p.nbr - 1;
  const float* unit_rec = p.part + (int64_t)unit * rec_per_unit * kBWaves * RB::kRec;
  const __amdgpu_buffer_rsrc_t urec =
      make_rsrc(unit_rec + ((int64_t)rbase * kBWaves + rbl) * RB::kRec, (uint32_t)(nwg * kBWaves * RB::kRec * 4));
  constexpr uint32_t kOutOff = 16 * RB::kRows;
  float Mg = -INFINITY, Lg = 0.f, Lxg = 0.f;
  f32x4 og[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) og[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  // a batch keeps the records as loaded (bf16 outputs still packed, unpacked when merged): fewer
  // VGPRs, so more of the launch's waves are resident at once
  constexpr int kOutWords = TRAIN ? 4 : 2;       // 16-byte output pieces per record and lane
  for (int k0 = 0; k0 < nwg; k0 += kMBatch) {
    f32x4 sv[kMBatch], ow[kMBatch][kOutWords];
#pragma unroll
    for (int u = 0; u < kMBatch; ++u) {
      const uint32_t rec = (uint32_t)(k0 + u) * kBWaves * RB::kRec * 4;
      const bool ok = k0 + u < nwg;
      sv[u] = ok ? load16_coherent(urec, rec + 16 * (16 * nt + lr)) : f32x4{-INFINITY, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < kOutWords; ++i) {
        const uint32_t piece = TRAIN ? (uint32_t)(nt * 8 + 4 * dh + i) : (uint32_t)(nt * 4 + 2 * dh + i);
        ow[u][i] = ok ? load16_coherent(urec, rec + kOutOff + 16 * (piece * kWave + lane)) : f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
#pragma unroll
    for (int u = 0; u < kMBatch; ++u) {
      if (k0 + u >= nwg) break;
      f32x4 ov[4];
      if constexpr (TRAIN) {
#pragma unroll
        for (int i = 0; i < 4; ++i) ov[i] = ow[u][i];
      } else {
#pragma unroll
        for (int k = 0; k < 2; ++k) unpack_record_bf16(as_u32x4(ow[u][k]), ov[2 * k], ov[2 * k + 1]);
      }
      const float mb = fmaxf(Mg, sv[u][0]);
      const float mbu = mb == -INFINITY ? 0.f : mb;
      const float sc = exp2f(Mg - mbu), wt = exp2f(sv[u][0] - mbu);
      Lg = Lg * sc + wt * sv[u][1];
      Lxg = Lxg * sc + wt * sv[u][2];
#pragma unroll
      for (int i = 0; i < 4; ++i) og[i] = og[i] * sc + ov[i] * wt;
      Mg = mb;
    }
  }
  // rows 16*nt + lane%16 of row block rb; register r of d-tile 4*dh + i holds d = 32*lg + 16*dh + 4*i + r
  const int nrow = rb * RB::kRows + 16 * nt + lr;
  if (nrow >= p.R) return;
  const int64_t view_rows = (int64_t)p.S * p.nq * p.Hq;
  const bool gb = b < p.V;
  uint16_t* out = gb ? p.out_g + (int64_t)b * view_rows * kD : p.out_f;
  float* lse = gb ? (p.lse_g ? p.lse_g + (int64_t)b * view_rows : nullptr) : p.lse_f;
  float* out32 = gb ? (p.o32_g ? p.o32_g + (int64_t)b * view_rows * kD : nullptr) : p.o32_f;
  const int j = nrow / p.G, h = g * p.G + nrow % p.G;
  const int64_t orow = ((int64_t)s * p.nq + j) * p.Hq + h;
  const float inv = Lg > 0.f ? 1.f / Lg : 0.f;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const f32x4 a = og[2 * k] * inv, c = og[2 * k + 1] * inv;
    const u32x4 wv = {pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3]), pack_bf16x2(c[0], c[1]),
                      pack_bf16x2(c[2], c[3])};
    const int d0 = 32 * lg + 16 * dh + 8 * k;
    *reinterpret_cast<u32x4*>(out + orow * kD + d0) = wv;
    if (TRAIN && out32) {
      *reinterpret_cast<f32x4*>(out32 + orow * kD + d0) = a;
      *reinterpret_cast<f32x4*>(out32 + orow * kD + d0 + 4) = c;
    }
  }
  if (lse && lg == 0 && dh == 0) lse[orow] = Lxg > 0.f ? (Mg + __log2f(Lxg)) * kLn2 : -INFINITY;
}

}  // namespace

// Counts held in int fields saturate at 2^30: the callers reject such shapes after planning (too many
// work units or workgroups), and the products formed from them stay inside int64.
static int sat_count(int64_t x) { return x > (int64_t(1) << 30) ? (1 << 30) : (int)x; }

AttnPlan plan_attn(int S, int Hkv, int Hq, int nq, int num_views, int ld_idx, int max_L, bool with_full, bool paged,
                   bool train, int page_size) {
  AttnPlan pl{};
  const int G = Hq / Hkv;
  pl.R = sat_count((int64_t)nq * G);
  pl.nt = pl.R <= 16 ? 1 : 2;
  const int rows = 16 * pl.nt;
  pl.n_rb = (pl.R + rows - 1) / rows;
  // several 32-row blocks share the K/V stream in block mode; the training outputs (fp32 output,
  // two-term weights) exist only there
  pl.block = pl.n_rb >= 2 || train;
  pl.n_rg = pl.block ? (pl.n_rb + kBWaves - 1) / kBWaves : pl.n_rb;
  pl.counter_bytes = BD_WS_COUNTER_BYTES;   // fixed: scratch of any call never lands on a counter
  if (pl.block) {
    // workgroups per (sequence, KV head, row group) unit, each taking an equal share of the unit's
    // key stream: enough to fill the CUs once, and enough that no share (rounded up to whole tiles)
    // overflows the slot table
    pl.units = sat_count((int64_t)S * Hkv * pl.n_rg);
    pl.nbr = sat_count((int64_t)num_views + (with_full ? 1 : 0));
    if (pl.nbr > kBMaxPieces) {      // more branches than a range holds pieces: not launchable
      pl.nblk = -1;
      pl.ws_bytes = pl.counter_bytes;
      return pl;
    }
    const int64_t stream_max = (int64_t)num_views * ld_idx + (with_full ? max_L : 0);
    int64_t nw = (kTargetBlocks + pl.units - 1) / pl.units;
    const int64_t nw_table = stream_cut_min_workgroups<kWGather, kWFull>(stream_max, kMaxSplitKeys);
    if (nw < nw_table) nw = nw_table;
    if (nw < 1) nw = 1;
    pl.nW = (int)nw;
    const int64_t blocks = (int64_t)pl.units * nw;
    pl.nblk = blocks > INT32_MAX ? -1 : (int)blocks;
    const size_t records = (size_t)pl.units * (nw + pl.nbr - 1) * kBWaves;   // one per piece and row block
    pl.record_bytes = nw > 1 ? align256(sizeof(float) * attn_record_floats(2) * records) : 0;
    pl.ws_bytes = pl.counter_bytes + pl.record_bytes;
    return pl;
  }
  pl.units_g = sat_count((int64_t)num_views * S * Hkv * pl.n_rg);
  pl.units_f = with_full ? sat_count((int64_t)S * Hkv * pl.n_rg) : 0;
  constexpr int64_t kStep = kWaves * kTile;       // one tile per wave of the split kernel
  auto round_up = [](int64_t x, int64_t m) { return (x + m - 1) / m * m; };
  const int64_t work = (int64_t)pl.units_g * ld_idx + (int64_t)pl.units_f * max_L;
  const int64_t g_all = round_up(ld_idx > 0 ? ld_idx : 1, kStep), f_all = round_up(max_L > 0 ? max_L : 1, kStep);
  // keys per split: the smallest multiple of kStep from work/kTargetBlocks up that keeps the
  // launch to one workgroup per CU (every kernel here holds one workgroup per CU), so no second
  // wave of workgroups forms a tail.  The gathered splits are bound by the slot table, and so is
  // the full branch of a paged cache; the full branch over a contiguous cache computes its row
  // offsets and is not.
  int64_t kps = round_up((work + kTargetBlocks - 1) / kTargetBlocks, kStep);
  if (kps < kStep) kps = kStep;
  // with more units than target workgroups no split count reaches the target: the search below
  // would end at one split per unit, so it starts there
  if ((int64_t)pl.units_g + pl.units_f > kTargetBlocks) {
    const int64_t all = g_all > f_all ? g_all : f_all;
    if (kps < all) kps = all;
  }
  // the paged full branch: its table holds kSlotCap entries, one per key, or one per page when pages
  // hold whole 16-key sub-tiles (a split of kf keys spans at most kf / page_size + 2 pages); key
  // indices below 2^26 keep the kernel's page division in its exact range
  pl.page_arith = paged && page_size > 0 && page_size % 16 == 0 && max_L <= (1 << 26) - 64;
  const int64_t kf_cap = pl.page_arith ? ((int64_t)(kSlotCap - 2) * page_size) / kStep * kStep : kMaxSplitKeys;
  int64_t kg, kf, blocks;
  for (;;) {
    kg = kps < g_all ? kps : g_all;
    if (kg > kMaxSplitKeys) kg = kMaxSplitKeys;
    kf = kps < f_all ? kps : f_all;
    if (paged && kf > kf_cap) kf = kf_cap;
    blocks = (int64_t)pl.units_g * ((g_all + kg - 1) / kg) + (int64_t)pl.units_f * ((f_all + kf - 1) / kf);
    if (blocks <= kTargetBlocks || (kps >= g_all && kps >= f_all)) break;
    kps += kStep;
  }
  pl.kps_g = (int)kg;
  pl.kps_f = (int)kf;
  pl.nsplit_g = ld_idx > 0 ? (int)((ld_idx + kg - 1) / kg) : 1;
  pl.nsplit_f = max_L > 0 ? (int)((max_L + kf - 1) / kf) : 1;
  blocks = (int64_t)pl.units_g * pl.nsplit_g + (int64_t)pl.units_f * pl.nsplit_f;
  pl.nblk = blocks > INT32_MAX ? -1 : (int)blocks;
  // group counters per unit for the two-level merge (units of more than kMergeGroup splits)
  auto groups = [](int n) { return n > kMergeGroup ? (n + kMergeGroup - 1) / kMergeGroup : 0; };
  const int gg = pl.units_g ? groups(pl.nsplit_g) : 0, gf = pl.units_f ? groups(pl.nsplit_f) : 0;
  pl.ngrp = gg > gf ? gg : gf;
  const bool split = (pl.units_g && pl.nsplit_g > 1) || (pl.units_f && pl.nsplit_f > 1);
  pl.record_bytes = split ? align256(sizeof(float) * attn_record_floats(pl.nt) * (size_t)blocks) : 0;
  pl.ws_bytes = pl.counter_bytes + pl.record_bytes;
  return pl;
}

template <int NT, bool PAGED>
static hipError_t launch_nt(const AttnParams& p, int nblocks, bool two_level, hipStream_t stream) {
  if (two_level) hipLaunchKernelGGL((attn_kernel<NT, PAGED, true>), dim3(nblocks), dim3(kThreads), 0, stream, p);
  else hipLaunchKernelGGL((attn_kernel<NT, PAGED, false>), dim3(nblocks), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_attn(const AttnParams& args, const AttnPlan& pl, bool paged, hipStream_t stream) {
  AttnParams p = args;
  p.nblk = pl.nblk;
  if (pl.block) {
    const bool train = p.o32_g || p.o32_f;
    if (train) {
      if (paged) hipLaunchKernelGGL((block_kernel<true, true>), dim3(pl.nblk), dim3(kBThreads), 0, stream, p);
      else hipLaunchKernelGGL((block_kernel<false, true>), dim3(pl.nblk), dim3(kBThreads), 0, stream, p);
    } else {
      if (paged) hipLaunchKernelGGL((block_kernel<true, false>), dim3(pl.nblk), dim3(kBThreads), 0, stream, p);
      else hipLaunchKernelGGL((block_kernel<false, false>), dim3(pl.nblk), dim3(kBThreads), 0, stream, p);
    }
    if (pl.nW > 1) {                               // some branch may be split: merge its records
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      // one workgroup per (unit, branch, row block): its four waves take the (row tile, d half) pairs
      const int64_t mblocks = (int64_t)pl.units * pl.nbr * kBWaves;
      if (train) hipLaunchKernelGGL((block_merge_kernel<true>), dim3((unsigned)mblocks), dim3(4 * kWave), 0, stream, p);
      else hipLaunchKernelGGL((block_merge_kernel<false>), dim3((unsigned)mblocks), dim3(4 * kWave), 0, stream, p);
    }
    return hipGetLastError();
  }
  const bool two = pl.ngrp > 0;
  if (pl.nt == 1)
    return paged ? launch_nt<1, true>(p, pl.nblk, two, stream) : launch_nt<1, false>(p, pl.nblk, two, stream);
  return paged ? launch_nt<2, true>(p, pl.nblk, two, stream) : launch_nt<2, false>(p, pl.nblk, two, stream);
}

size_t attn_ws_bytes(int S, int Hkv, int Hq, int nq, int num_views, int ld_idx, int max_L, bool with_full,
                     bool train_capable) {
  size_t best = 0;   // over the variants that can launch; 0 if none can
  for (int paged = 0; paged < 2; ++paged)
    for (int train = 0; train <= (train_capable ? 1 : 0); ++train) {
      const AttnPlan pl = plan_attn(S, Hkv, Hq, nq, num_views, ld_idx, max_L, with_full, paged != 0, train != 0);
      if (pl.nblk < 0) continue;
      best = pl.ws_bytes > best ? pl.ws_bytes : best;
    }
  return best;
}

size_t attn_record_floats(int nt) { return nt == 1 ? RowBlock<1>::kRec : RowBlock<2>::kRec; }

}  // namespace bd
