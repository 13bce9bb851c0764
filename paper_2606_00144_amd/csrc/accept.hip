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
    for (int c = c0 + 4 * tid; c < c1; c += 4 * kThreads) {
      if (c + 4 <= c1) {
        const f32x4 x = *reinterpret_cast<const f32x4*>(row + c);
        best = umax64(best, pack_key(x[0], c));
        best = umax64(best, pack_key(x[1], c + 1));
        best = umax64(best, pack_key(x[2], c + 2));
        best = umax64(best, pack_key(x[3], c + 3));
      } else {
        for (int e = c; e < c1; ++e) best = umax64(best, pack_key(row[e], e));
      }
    }
  } else {
    for (int c = c0 + tid; c < c1; c += kThreads) best = umax64(best, pack_key(row[c], c));
  }
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) best = umax64(best, shfl_xor_u64(best, m));
  if ((tid & 63) == 0) red[tid >> 6] = best;
  __syncthreads();

  const int per_seq = rows * p.nsplit;
  if (per_seq > 1) {
    if (tid == 0) {
      uint64_t bb = red[0];
      for (int w = 1; w < kThreads / kWave; ++w) bb = umax64(bb, red[w]);
      store_coherent(p.part + (int64_t)rs * p.nsplit + split, bb);
      wait_vmem();
      last = arrive(&p.counters[s], (uint32_t)per_seq);
    }
    __syncthreads();
    if (!last) return;
    // merge: thread i < rows takes row i (rows <= 64 is checked on the host)
    if (tid < rows) {
      const uint64_t* pr = p.part + ((int64_t)s * rows + tid) * p.nsplit;
      uint64_t bb = 0;
      for (int sp = 0; sp < p.nsplit; ++sp) bb = umax64(bb, load_coherent(pr + sp));
      rowbest[tid] = bb;
    }
  } else if (tid == 0) {
    uint64_t bb = red[0];
    for (int w = 1; w < kThreads / kWave; ++w) bb = umax64(bb, red[w]);
    rowbest[0] = bb;
  }
  __syncthreads();
  if (tid == 0) {
    int k = 0;
    while (k < p.gamma && p.draft[(int64_t)s * p.gamma + k] == (int32_t)(0xFFFFFFFFu - (uint32_t)rowbest[k])) ++k;
    p.accept_out[s] = k;
    if (p.bonus_out) p.bonus_out[s] = (int32_t)(0xFFFFFFFFu - (uint32_t)rowbest[k]);
    if (per_seq > 1) reset_counter(&p.counters[s]);
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
  if (want > max_split) want = max_split;
  if (want < 1) want = 1;
  int64_t chunk = (vocab + want - 1) / want;
  chunk = (chunk + 3) & ~int64_t(3);
  pl.chunk = (int)chunk;
  pl.nsplit = (int)((vocab + chunk - 1) / chunk);
  pl.counter_bytes = BD_WS_COUNTER_BYTES;
  pl.ws_bytes = pl.counter_bytes + align256(sizeof(uint64_t) * (size_t)rows * pl.nsplit);
  return pl;
}

hipError_t launch_accept(const AcceptParams& p, hipStream_t stream) {
  const int nblocks = p.S * (p.gamma + 1) * p.nsplit;
  hipLaunchKernelGGL(accept_kernel, dim3(nblocks), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace bd
