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

namespace bd {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * kWave;
constexpr int kTile = 32;                      // keys per wave iteration
constexpr int64_t kTargetBlocks = 512;         // workgroups per launch the splits aim for
constexpr float kLn2 = 0.6931471805599453f;

template <int NT>
struct RowBlock {
  static constexpr int kRows = 16 * NT;
  static constexpr int kRec = kRows * (3 + kD);   // floats of one partial record: m, l, lx, o[128]
};

// LDS scratch of one workgroup.
template <int NT>
struct AttnSmem {
  alignas(16) float o[kWaves][16 * NT][kD];     // per-wave unnormalised outputs
  float m[kWaves][16 * NT];
  float l[kWaves][16 * NT];
  float lx[kWaves][16 * NT];
  int32_t sidx[kMaxGatherSplit];    // gathered positions of this split
  int32_t last;
};

// Resolve the key position of slot u (0..31) of a tile starting at slot b.
struct KeySlots {
  bool gather;
  const int32_t* sidx;   // LDS copy of idx[e_begin .. e_end)
  int e_begin, e_end;    // slot range of this split
  int L;
  __device__ int pos(int slot) const {   // absolute slot -> position or -1
    if (slot >= e_end) return -1;
    const int t = gather ? sidx[slot - e_begin] : slot;
    return (t >= 0 && t < L) ? t : -1;
  }
};

template <int NT, bool PAGED>
struct TileRegs {
  u32x4 k[2][4];     // [key subtile][k-step]: 16 keys x 64 B per lane group
  u32x4 v[8];        // 8 key rows x 16 B
  int tpos[8];       // positions of the 8 score slots (-1 = absent)
};

template <int NT, bool PAGED>
__device__ inline void load_tile(TileRegs<NT, PAGED>& T, const KvView& kv, const KeySlots& ks, int s, int g,
                                 int slot0, int lane) {
  const int lg = lane >> 4, lr = lane & 15;
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) {
    const int t = ks.pos(slot0 + 16 * sub + lr);
    int64_t off = t >= 0 ? row_offset<PAGED>(kv, s, g, t) : -1;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (off >= 0) T.k[sub][j] = load16(kv.k + off + 32 * lg + 8 * j);
      else T.k[sub][j] = u32x4{0u, 0u, 0u, 0u};
    }
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int slot = 16 * (i >> 2) + 4 * lg + (i & 3);
    const int t = ks.pos(slot0 + slot);
    int64_t off = t >= 0 ? row_offset<PAGED>(kv, s, g, t) : -1;
    T.tpos[i] = off >= 0 ? t : -1;
    if (off >= 0) T.v[i] = load16(kv.v + off + 8 * lr);
    else T.v[i] = u32x4{0u, 0u, 0u, 0u};
  }
}

// Transposed V operand for d-tile dt: slot i holds V[key slot i][8*(lane%16) + dt].
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

template <int NT>
struct RowState {
  f32x4 o[NT][8];     // O^T[d-tile][row tile]
  float m[NT];        // running max (log2 domain), shared by the 4 lane groups
  float l[NT];        // running sum of the bf16-rounded weights the PV product uses (normaliser)
  float lx[NT];       // running sum of the unrounded weights (log-sum-exp); both this lane's keys only
};

template <int NT, bool PAGED>
__device__ inline void tile_step(RowState<NT>& st, const TileRegs<NT, PAGED>& T, const bf16x8 (&qop)[NT][4],
                                 const int (&rowpos)[NT], float scale_log2) {
  // scores S^T for 32 keys x 16*NT rows
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

  bf16x8 pop[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float sv[8];
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float x = sacc[i >> 2][nt][i & 3] * scale_log2;
      const bool vis = T.tpos[i] >= 0 && T.tpos[i] <= rowpos[nt];
      sv[i] = vis ? x : -INFINITY;
      mx = fmaxf(mx, sv[i]);
    }
    mx = fmaxf(mx, shfl_xor_f(mx, 16));
    mx = fmaxf(mx, shfl_xor_f(mx, 32));
    const float mnew = fmaxf(st.m[nt], mx);
    const float muse = mnew == -INFINITY ? 0.f : mnew;
    const float alpha = exp2f(st.m[nt] - muse);
    float psum = 0.f, pxsum = 0.f;
    u32x4 pw;
#pragma unroll
    for (int i = 0; i < 8; i += 2) {
      // the sum uses the bf16-rounded weights that the PV product sees
      const float p0 = exp2f(sv[i] - muse), p1 = exp2f(sv[i + 1] - muse);
      const uint32_t w = pack_bf16x2(p0, p1);
      pxsum += p0 + p1;
      psum += bf16_lo(w) + bf16_hi(w);
      pw[i >> 1] = w;
    }
    pop[nt] = as_bf16x8(pw);
    st.l[nt] = st.l[nt] * alpha + psum;
    st.lx[nt] = st.lx[nt] * alpha + pxsum;
    st.m[nt] = mnew;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) st.o[nt][dt] *= alpha;
  }

#pragma unroll
  for (int dt = 0; dt < 8; ++dt) {
    const bf16x8 vt = vt_operand(T.v, dt);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
      st.o[nt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vt, pop[nt], st.o[nt][dt], 0, 0, 0);
  }
}

template <int NT, bool PAGED>
__global__ __launch_bounds__(kThreads) void attn_kernel(AttnParams p) {
  using RB = RowBlock<NT>;
  __shared__ AttnSmem<NT> sm;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int lg = lane >> 4, lr = lane & 15;

  // ---- which (kind, unit, split) this workgroup owns
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const bool gather = bid < p.nblk_g;
  const int local = gather ? bid : bid - p.nblk_g;
  const int nsplit = gather ? p.nsplit_g : p.nsplit_f;
  const int kps = gather ? p.kps_g : p.kps_f;
  const int rb = local % p.n_rb;
  const int rest = local / p.n_rb;
  const int split = rest % nsplit;
  const int pair = rest / nsplit;          // gather: (view, s, g); full: (s, g)
  const int g = pair % p.Hkv;
  const int vs = pair / p.Hkv;             // gather: view*S + s; full: s
  const int s = gather ? vs % p.S : vs;
  const int view = gather ? vs / p.S : 0;
  const int unit = gather ? pair * p.n_rb + rb : p.units_g + pair * p.n_rb + rb;

  const int L = seq_len(p.kv, s);
  int n_keys;
  const int32_t* idx_row = nullptr;
  if (gather) {
    idx_row = p.idx + ((int64_t)vs * p.Hkv + g) * p.ld_idx;
    int n = p.nsel[vs];
    n_keys = n < 0 ? 0 : (n > p.ld_idx ? p.ld_idx : n);
  } else {
    n_keys = L;
  }
  const int e_begin = split * kps;
  int e_end = e_begin + kps;
  if (e_end > n_keys) e_end = n_keys;

  if (gather) {
    for (int i = tid; i < kps; i += kThreads) {
      const int e = e_begin + i;
      sm.sidx[i] = e < e_end ? idx_row[e] : -1;
    }
    __syncthreads();
  }
  KeySlots ks{gather, sm.sidx, e_begin, e_end, L};

  // ---- query rows of this lane: row n = rb*RB + 16*nt + lane%16
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

  RowState<NT> st;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    st.m[nt] = -INFINITY;
    st.l[nt] = 0.f;
    st.lx[nt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) st.o[nt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // ---- stream this wave's tiles (tile w, w+4, ...), one tile of loads in flight ahead
  const int ntiles = e_end > e_begin ? (e_end - e_begin + kTile - 1) / kTile : 0;
  if (wave < ntiles) {
    TileRegs<NT, PAGED> ta, tb;
    load_tile<NT, PAGED>(ta, p.kv, ks, s, g, e_begin + kTile * wave, lane);
    int it = wave;
    while (true) {
      const int nx = it + kWaves;
      if (nx < ntiles) load_tile<NT, PAGED>(tb, p.kv, ks, s, g, e_begin + kTile * nx, lane);
      tile_step<NT, PAGED>(st, ta, qop, rowpos, p.scale_log2);
      if (nx >= ntiles) break;
      const int nx2 = nx + kWaves;
      if (nx2 < ntiles) load_tile<NT, PAGED>(ta, p.kv, ks, s, g, e_begin + kTile * nx2, lane);
      tile_step<NT, PAGED>(st, tb, qop, rowpos, p.scale_log2);
      if (nx2 >= ntiles) break;
      it = nx2;
    }
  }

  // ---- wave state -> LDS: row r = 16*nt + lane%16; lane group lg holds d in [32lg, 32lg+32)
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float l = st.l[nt], lx = st.lx[nt];
    l += shfl_xor_f(l, 16);
    l += shfl_xor_f(l, 32);
    lx += shfl_xor_f(lx, 16);
    lx += shfl_xor_f(lx, 32);
    const int r = 16 * nt + lr;
    if (lg == 0) {
      sm.m[wave][r] = st.m[nt];
      sm.l[wave][r] = l;
      sm.lx[wave][r] = lx;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float* dst = &sm.o[wave][r][32 * lg + 8 * i];
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
  for (int w = 0; w < kWaves; ++w) M = fmaxf(M, sm.m[w][r]);
  const float Muse = M == -INFINITY ? 0.f : M;
  float Lsum = 0.f, Lx = 0.f, acc[kPerThread];
#pragma unroll
  for (int e = 0; e < kPerThread; ++e) acc[e] = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const float wt = exp2f(sm.m[w][r] - Muse);
    Lsum += wt * sm.l[w][r];
    Lx += wt * sm.lx[w][r];
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) acc[e] += wt * sm.o[w][r][d0 + e];
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

  // ---- publish this split's partial record (rows that exist only); the last split merges them
  float* rec_base = p.part + (gather ? 0 : (int64_t)p.units_g * p.nsplit_g * RB::kRec);
  const int unit_local = gather ? unit : unit - p.units_g;
  float* rec = rec_base + ((int64_t)unit_local * nsplit + split) * RB::kRec;
  if (row_valid) {
    if (d0 == 0) {
      store_coherent(rec + 3 * r, M);
      store_coherent(rec + 3 * r + 1, Lsum);
      store_coherent(rec + 3 * r + 2, Lx);
    }
    float* ro = rec + 3 * RB::kRows + r * kD + d0;
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) store_coherent(ro + e, acc[e]);
  }
  wait_vmem();
  __syncthreads();
  if (tid == 0) sm.last = arrive(&p.counters[unit], (uint32_t)nsplit);
  __syncthreads();
  if (!sm.last) return;
  if (tid == 0) reset_counter(&p.counters[unit]);   // ready for the next call
  if (!row_valid) return;

  const float* urec = rec_base + (int64_t)unit_local * nsplit * RB::kRec;
  float Mg = -INFINITY;
  for (int sp = 0; sp < nsplit; ++sp) Mg = fmaxf(Mg, load_coherent(urec + (int64_t)sp * RB::kRec + 3 * r));
  const float Mgu = Mg == -INFINITY ? 0.f : Mg;
  float Lg = 0.f, Lxg = 0.f, ag[kPerThread];
#pragma unroll
  for (int e = 0; e < kPerThread; ++e) ag[e] = 0.f;
  for (int sp = 0; sp < nsplit; ++sp) {
    const float* rs = urec + (int64_t)sp * RB::kRec;
    const float wt = exp2f(load_coherent(rs + 3 * r) - Mgu);
    Lg += wt * load_coherent(rs + 3 * r + 1);
    Lxg += wt * load_coherent(rs + 3 * r + 2);
    const float* os = rs + 3 * RB::kRows + r * kD + d0;
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) ag[e] += wt * load_coherent(os + e);
  }
  write_final(Mg, Lg, Lxg, ag);
}

}  // namespace

AttnPlan plan_attn(int S, int Hkv, int Hq, int nq, int num_views, int ld_idx, int max_L, bool with_full) {
  AttnPlan pl{};
  const int G = Hq / Hkv;
  pl.R = nq * G;
  pl.nt = pl.R <= 16 ? 1 : 2;
  const int rows = 16 * pl.nt;
  pl.n_rb = (pl.R + rows - 1) / rows;
  pl.units_g = num_views * S * Hkv * pl.n_rb;
  pl.units_f = with_full ? S * Hkv * pl.n_rb : 0;
  constexpr int64_t kStep = kWaves * kTile;       // one tile per wave
  auto round_up = [](int64_t x, int64_t m) { return (x + m - 1) / m * m; };
  const int64_t work = (int64_t)pl.units_g * ld_idx + (int64_t)pl.units_f * max_L;
  int64_t kps = round_up((work + kTargetBlocks - 1) / kTargetBlocks, kStep);
  if (kps < kStep) kps = kStep;
  int64_t kg = kps < round_up(ld_idx > 0 ? ld_idx : 1, kStep) ? kps : round_up(ld_idx > 0 ? ld_idx : 1, kStep);
  if (kg > kMaxGatherSplit) kg = kMaxGatherSplit;
  int64_t kf = kps < round_up(max_L > 0 ? max_L : 1, kStep) ? kps : round_up(max_L > 0 ? max_L : 1, kStep);
  pl.kps_g = (int)kg;
  pl.kps_f = (int)kf;
  pl.nsplit_g = ld_idx > 0 ? (int)((ld_idx + kg - 1) / kg) : 1;
  pl.nsplit_f = max_L > 0 ? (int)((max_L + kf - 1) / kf) : 1;
  const int64_t blocks = (int64_t)pl.units_g * pl.nsplit_g + (int64_t)pl.units_f * pl.nsplit_f;
  pl.nblk = (int)blocks;
  pl.counter_bytes = BD_WS_COUNTER_BYTES;   // fixed: scratch of any call never lands on a counter
  const bool split = (pl.units_g && pl.nsplit_g > 1) || (pl.units_f && pl.nsplit_f > 1);
  pl.record_bytes = split ? align256(sizeof(float) * attn_record_floats(pl.nt) * (size_t)blocks) : 0;
  pl.ws_bytes = pl.counter_bytes + pl.record_bytes;
  return pl;
}

template <int NT, bool PAGED>
static hipError_t launch_nt(const AttnParams& p, int nblocks, hipStream_t stream) {
  hipLaunchKernelGGL((attn_kernel<NT, PAGED>), dim3(nblocks), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_attn(const AttnParams& p, int nt, bool paged, int nblocks, hipStream_t stream) {
  if (nt == 1) return paged ? launch_nt<1, true>(p, nblocks, stream) : launch_nt<1, false>(p, nblocks, stream);
  return paged ? launch_nt<2, true>(p, nblocks, stream) : launch_nt<2, false>(p, nblocks, stream);
}

size_t attn_record_floats(int nt) { return nt == 1 ? RowBlock<1>::kRec : RowBlock<2>::kRec; }

}  // namespace bd
