// Greedy acceptance over verifier logits (Eq. 3; Alg. 2 accept and bonus token).
//
// Every (sequence, row, vocab chunk) workgroup scans its chunk once with
// 16-byte loads.  A thread keeps the first maximum of its own elements (it
// visits them in increasing index order, so a strict compare keeps the lowest
// index); the workgroup then reduces packed keys (order(value) << 32) | ~index,
// which are maximal exactly at the lowest-index maximum, and max-combines its
// key into the row's slot with a device-scope atomic.  The last chunk of a row
// to finish counts the row done; the last row of a sequence reads its row
// maxima and counts the leading drafts that equal the verifier's greedy tokens.

#include "bd_common.hpp"
#include "bd_kernels.hpp"

namespace bd {
namespace {

constexpr int kThreads = 256;
constexpr int kTargetBlocks = 768;
constexpr int kUnroll = 8;          // float4 loads in flight per thread

__device__ inline uint64_t pack_key(float v, int idx) {
  return ((uint64_t)float_order_key(v) << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)idx);
}
__device__ inline int key_index(uint64_t k) { return (int)(0xFFFFFFFFu - (uint32_t)k); }

__device__ inline uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }

__device__ inline uint64_t shfl_xor_u64(uint64_t x, int m) {
  const int src = (int)(threadIdx.x ^ m) & (kWave - 1);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_ds_bpermute(src << 2, (int)(uint32_t)x);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_ds_bpermute(src << 2, (int)(uint32_t)(x >> 32));
  return ((uint64_t)hi << 32) | lo;
}

// Every kernel argument requested at entry, so the argument lines cost one memory round trip (the
// compiler would otherwise fetch each where it is first used).  The statements touch no memory and
// return 0, which the caller adds to its block index.
__device__ inline int fetch_args(const AcceptParams& p) {
  int z;
  asm("s_mov_b32 %0, 0" : "=s"(z) : "s"(p.logits), "s"(p.row_stride), "s"(p.draft), "s"(p.S), "s"(p.gamma),
      "s"(p.vocab), "s"(p.nsplit), "s"(p.chunk), "s"(p.vec4), "s"(p.accept_out), "s"(p.bonus_out),
      "s"(p.argmax_out), "s"(p.counters), "s"(p.nblk));
  return z;
}

__global__ __launch_bounds__(kThreads) void accept_kernel(AcceptParams p) {
  __shared__ uint64_t red[kThreads / kWave];
  __shared__ uint64_t rowbest[64];
  __shared__ int32_t last;
  const int tid = threadIdx.x;
  const int rows = p.gamma + 1;
  const int nrows = p.S * rows;
  const int b = xcd_remap(blockIdx.x + fetch_args(p), p.nblk);
  const int rs = div_small(b, p.nsplit);    // s * rows + i
  const int split = b - rs * p.nsplit;
  const int s = div_small(rs, rows);
  // this sequence's drafts, loaded with the first loads (only the sequence's last workgroup uses them)
  const int my_draft = tid < p.gamma ? p.draft[(int64_t)s * p.gamma + tid] : -1;
  uint32_t* seq_counter = counter_line(p.counters, s);
  uint32_t* row_counter = counter_line(p.counters, p.S + rs);
  auto row_slot = [&](int r) { return reinterpret_cast<uint64_t*>(counter_line(p.counters, p.S + nrows + r)); };

  const float* row = p.logits + (int64_t)rs * p.row_stride;
  const int c0 = split * p.chunk;
  int c1 = c0 + p.chunk;
  if (c1 > p.vocab) c1 = p.vocab;

  // first maximum of this thread's elements (all finite by contract; a thread whose elements are
  // all -inf reports its first one)
  float bv = -INFINITY;
  int bi = -1, first = -1;
  if (p.vec4) {
    // each thread's float4 loads of a round are all issued before any is reduced
    for (int base = c0 + 4 * tid; base < c1; base += 4 * kThreads * kUnroll) {
      f32x4 x[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int c = base + u * 4 * kThreads;
        // non-temporal: the logits are read once per step, after verify has streamed the caches
        x[u] = c + 4 <= c1 ? __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(row + c)) : f32x4{0.f, 0.f, 0.f, 0.f};
      }
      if (first < 0) first = base;
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int c = base + u * 4 * kThreads;
        if (c + 4 <= c1) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const bool gt = x[u][e] > bv;
            bv = gt ? x[u][e] : bv;
            bi = gt ? c + e : bi;
          }
        } else {
          for (int e = c; e < c1; ++e) {
            const float v = row[e];
            if (v > bv) { bv = v; bi = e; }
          }
        }
      }
    }
  } else {
    for (int c = c0 + tid; c < c1; c += kThreads) {
      if (first < 0) first = c;
      const float v = row[c];
      if (v > bv) { bv = v; bi = c; }
    }
  }
  uint64_t best = bi >= 0 ? pack_key(bv, bi) : (first >= 0 ? pack_key(-INFINITY, first) : 0ull);
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) best = umax64(best, shfl_xor_u64(best, m));
  if ((tid & 63) == 0) red[tid >> 6] = best;
  __syncthreads();

  // Two-level completion keeps the arrivals per counter few: nsplit chunks per row counter,
  // gamma+1 rows per sequence counter.
  if (tid == 0) {
    uint64_t bb = red[0];
    for (int w = 1; w < kThreads / kWave; ++w) bb = umax64(bb, red[w]);
    bool row_done = true;
    if (p.nsplit > 1) {
      atomic_max_coherent(row_slot(rs), bb);
      wait_vmem();
      row_done = arrive(row_counter, (uint32_t)p.nsplit);
      if (row_done) reset_counter(row_counter);
    } else {
      store_coherent(row_slot(rs), bb);
      wait_vmem();
    }
    last = row_done && (rows == 1 || arrive(seq_counter, (uint32_t)rows));
  }
  __syncthreads();
  if (!last) return;
  if (tid < rows) {
    uint64_t* slot = row_slot(s * rows + tid);
    rowbest[tid] = load_coherent(slot);
    store_coherent(slot, 0ull);   // the slots start from zero in the next call
  }
  __syncthreads();
  // accepted drafts: the leading run of matches, one ballot over the gamma comparisons (gamma <= 63,
  // so bit gamma is clear and the run ends there at the latest)
  if (tid < kWave) {
    const uint64_t key = tid < rows ? rowbest[tid] : 0ull;
    const uint64_t match = __builtin_amdgcn_ballot_w64(tid < p.gamma && my_draft == key_index(key));
    const int k = __builtin_ctzll(~match);
    if (tid == 0) {
      p.accept_out[s] = k;
      if (p.bonus_out) p.bonus_out[s] = key_index(rowbest[k]);
      if (rows > 1) reset_counter(seq_counter);
    }
    if (p.argmax_out && tid < rows) p.argmax_out[(int64_t)s * rows + tid] = key_index(key);
  }
}

}  // namespace

AcceptPlan plan_accept(int S, int gamma, int vocab) {
  AcceptPlan pl;
  const int64_t rows = (int64_t)S * (gamma + 1);
  int64_t want = (kTargetBlocks + rows - 1) / rows;
  const int64_t max_split = ((int64_t)vocab + 4 * kThreads - 1) / (4 * kThreads);   // >= 1024 floats per chunk
  const int64_t min_split = ((int64_t)vocab + 4 * kThreads * kUnroll - 1) / (4 * kThreads * kUnroll);   // one load round
  if (want > max_split) want = max_split;
  if (want < min_split) want = min_split;
  if (want < 1) want = 1;
  int64_t chunk = ((int64_t)vocab + want - 1) / want;
  chunk = (chunk + 3) & ~int64_t(3);
  pl.chunk = (int)chunk;
  pl.nsplit = (int)((vocab + chunk - 1) / chunk);
  pl.counter_bytes = BD_WS_COUNTER_BYTES;   // counters and row maxima live in the counter region
  pl.ws_bytes = pl.counter_bytes;
  return pl;
}

hipError_t launch_accept(const AcceptParams& p, hipStream_t stream) {
  AcceptParams a = p;
  a.nblk = p.S * (p.gamma + 1) * p.nsplit;
  hipLaunchKernelGGL(accept_kernel, dim3(a.nblk), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace bd
