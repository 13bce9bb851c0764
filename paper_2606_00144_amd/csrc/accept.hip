// Greedy acceptance over verifier logits (Eq. 3; Alg. 2 accept and bonus token).
//
// Every (sequence, row, vocab chunk) workgroup scans its chunk once with
// 16-byte loads and reduces (order key of the value, index) to the maximum,
// lower index winning ties: the packed key (order(value) << 32) | ~index is
// maximal exactly there.  The last workgroup of a sequence to finish (atomic
// counter) merges the chunk results of all gamma+1 rows and counts the
// leading drafts that equal the verifier's greedy tokens.

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

__device__ inline uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }

__device__ inline uint64_t shfl_xor_u64(uint64_t x, int m) {
  const int src = (int)(threadIdx.x ^ m) & (kWave - 1);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_ds_bpermute(src << 2, (int)(uint32_t)x);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_ds_bpermute(src << 2, (int)(uint32_t)(x >> 32));
  return ((uint64_t)hi << 32) | lo;
}

__global__ __launch_bounds__(kThreads) void accept_kernel(AcceptParams p) {
  __shared__ uint64_t red[kThreads / kWave];
  __shared__ uint64_t rowbest[64];
  __shared__ int32_t last;
  const int tid = threadIdx.x;
  const int rows = p.gamma + 1;
  const int b = xcd_remap(blockIdx.x, gridDim.x);
  const int split = b % p.nsplit;
  const int rs = b / p.nsplit;              // s * rows + i
  const int s = rs / rows;

  const float* row = p.logits + (int64_t)rs * p.row_stride;
  const int c0 = split * p.chunk;
  int c1 = c0 + p.chunk;
  if (c1 > p.vocab) c1 = p.vocab;

  uint64_t best = 0;
  if (p.vec4) {
    // each thread's float4 loads of the chunk are all issued before any is reduced
    for (int base = c0 + 4 * tid; base < c1; base += 4 * kThreads * kUnroll) {
      f32x4 x[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int c = base + u * 4 * kThreads;
        x[u] = c + 4 <= c1 ? *reinterpret_cast<const f32x4*>(row + c) : f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int c = base + u * 4 * kThreads;
        if (c + 4 <= c1) {
          best = umax64(best, pack_key(x[u][0], c));
          best = umax64(best, pack_key(x[u][1], c + 1));
          best = umax64(best, pack_key(x[u][2], c + 2));
          best = umax64(best, pack_key(x[u][3], c + 3));
        } else {
          for (int e = c; e < c1; ++e) best = umax64(best, pack_key(row[e], e));
        }
      }
    }
  } else {
    for (int c = c0 + tid; c < c1; c += kThreads) best = umax64(best, pack_key(row[c], c));
  }
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) best = umax64(best, shfl_xor_u64(best, m));
  if ((tid & 63) == 0) red[tid >> 6] = best;
  __syncthreads();

  // Two-level completion: the last chunk of a row merges that row (nsplit arrivals on the row's
  // counter), the last row of a sequence counts the accepted prefix (gamma+1 arrivals on the
  // sequence's counter).  Few arrivals per counter keep the atomics from serialising.
  __shared__ int32_t last_seq;
  if (p.nsplit > 1) {
    if (tid == 0) {
      uint64_t bb = red[0];
      for (int w = 1; w < kThreads / kWave; ++w) bb = umax64(bb, red[w]);
      store_coherent(p.part + (int64_t)rs * p.nsplit + split, bb);
      wait_vmem();
      last = arrive(&p.counters[p.S + rs], (uint32_t)p.nsplit);
    }
    __syncthreads();
    if (!last) return;
    if (tid < kWave) {   // one wave merges the row's chunks, 64 loads in flight per pass
      uint64_t bb = 0;
      const uint64_t* pr = p.part + (int64_t)rs * p.nsplit;
      for (int sp = tid; sp < p.nsplit; sp += kWave) bb = umax64(bb, load_coherent(pr + sp));
#pragma unroll
      for (int m = 1; m < kWave; m <<= 1) bb = umax64(bb, shfl_xor_u64(bb, m));
      if (tid == 0) {
        reset_counter(&p.counters[p.S + rs]);
        red[0] = bb;
      }
    }
    __syncthreads();
  } else if (tid == 0) {
    uint64_t bb = red[0];
    for (int w = 1; w < kThreads / kWave; ++w) bb = umax64(bb, red[w]);
    red[0] = bb;
  }
  // red[0] is the merged key of row rs; publish it and let the sequence's last row finish
  if (tid == 0) {
    store_coherent(p.rowbest + rs, red[0]);
    wait_vmem();
    last_seq = rows == 1 ? 1 : arrive(&p.counters[s], (uint32_t)rows);
  }
  __syncthreads();
  if (!last_seq) return;
  if (tid < rows) rowbest[tid] = load_coherent(p.rowbest + (int64_t)s * rows + tid);
  __syncthreads();
  if (tid == 0) {
    int k = 0;
    while (k < p.gamma && p.draft[(int64_t)s * p.gamma + k] == (int32_t)(0xFFFFFFFFu - (uint32_t)rowbest[k])) ++k;
    p.accept_out[s] = k;
    if (p.bonus_out) p.bonus_out[s] = (int32_t)(0xFFFFFFFFu - (uint32_t)rowbest[k]);
    if (rows > 1) reset_counter(&p.counters[s]);
  }
  if (p.argmax_out && tid < rows)
    p.argmax_out[(int64_t)s * rows + tid] = (int32_t)(0xFFFFFFFFu - (uint32_t)rowbest[tid]);
}

}  // namespace

AcceptPlan plan_accept(int S, int gamma, int vocab) {
  AcceptPlan pl;
  const int64_t rows = (int64_t)S * (gamma + 1);
  int64_t want = (kTargetBlocks + rows - 1) / rows;
  const int64_t max_split = (vocab + 4 * kThreads - 1) / (4 * kThreads);   // >= 1024 floats per chunk
  const int64_t min_split = (vocab + 4 * kThreads * kUnroll - 1) / (4 * kThreads * kUnroll);   // one load round
  if (want > max_split) want = max_split;
  if (want < min_split) want = min_split;
  if (want < 1) want = 1;
  int64_t chunk = (vocab + want - 1) / want;
  chunk = (chunk + 3) & ~int64_t(3);
  pl.chunk = (int)chunk;
  pl.nsplit = (int)((vocab + chunk - 1) / chunk);
  pl.counter_bytes = BD_WS_COUNTER_BYTES;
  pl.part_bytes = align256(sizeof(uint64_t) * (size_t)rows * pl.nsplit);
  pl.ws_bytes = pl.counter_bytes + pl.part_bytes + align256(sizeof(uint64_t) * (size_t)rows);
  return pl;
}

hipError_t launch_accept(const AcceptParams& p, hipStream_t stream) {
  const int nblocks = p.S * (p.gamma + 1) * p.nsplit;
  hipLaunchKernelGGL(accept_kernel, dim3(nblocks), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace bd
