// Top-1 cross-entropy of the drafter against the verifier's greedy targets
// (targets: Eq. 5; the summand of L_A and L_C: Eqs. 6-7), fused with the scan
// that finds the targets, and Cat(B, w) budget sampling (Sec. 3.4).
//
// Every (row, vocab chunk) workgroup reads its chunk of the student logits once
// (running max and sum of exponentials, in registers, 16-byte loads issued
// before use) and, when the teacher logits are given, its chunk of those (first
// maximum, as in the acceptance kernel).  A chunk's result is one 16-byte
// record; the last chunk of a row (device-scope counter) merges the records in
// chunk order, reads the student logit of the target and writes the loss.

#include "bd_common.hpp"
#include "bd_kernels.hpp"

namespace bd {
namespace {

constexpr int kThreads = 256;
constexpr int kTargetBlocks = 768;
constexpr int kUnroll = 12;         // float4 loads in flight per thread and row: a chunk in one round
constexpr float kLog2e = 1.4426950408889634f;

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

// (m, s) <- merge of two (max, sum of exp(x - max)) pairs
__device__ inline void merge_ms(float& m, float& s, float m2, float s2) {
  const float M = fmaxf(m, m2);
  if (M == -INFINITY) return;
  s = s * __builtin_amdgcn_exp2f((m - M) * kLog2e) + s2 * __builtin_amdgcn_exp2f((m2 - M) * kLog2e);
  m = M;
}

__global__ __launch_bounds__(kThreads) void ce_kernel(CeParams p) {
  __shared__ float red_m[kThreads / kWave], red_s[kThreads / kWave];
  __shared__ uint64_t red_k[kThreads / kWave];
  __shared__ int32_t last;
  const int tid = threadIdx.x;
  const int b = xcd_remap(blockIdx.x, gridDim.x);
  const int split = b % p.nsplit;
  const int r = b / p.nsplit;
  const float* srow = p.student + (int64_t)r * p.s_stride;
  const float* trow = p.teacher ? p.teacher + (int64_t)r * p.t_stride : nullptr;
  const int c0 = split * p.chunk;
  int c1 = c0 + p.chunk;
  if (c1 > p.vocab) c1 = p.vocab;

  float m = -INFINITY, s = 0.f;            // this thread's student elements
  float bv = -INFINITY;                    // this thread's first teacher maximum
  int bi = -1, first = -1;
  auto add_one = [&](float x, int c, float tv) {
    merge_ms(m, s, x, 1.f);
    if (first < 0) first = c;
    if (trow && tv > bv) { bv = tv; bi = c; }
  };
  if (p.vec4) {
    const int c1v = c0 + ((c1 - c0) & ~3);   // whole float4s; the rest below
    for (int base = c0 + 4 * tid; base < c1v; base += 4 * kThreads * kUnroll) {
      f32x4 xs[kUnroll], xt[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int c = base + u * 4 * kThreads;
        const bool ok = c < c1v;
        xs[u] = ok ? *reinterpret_cast<const f32x4*>(srow + c) : f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
        if (trow) xt[u] = ok ? *reinterpret_cast<const f32x4*>(trow + c) : f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
      }
      if (first < 0) first = base;
      float tm = -INFINITY;
#pragma unroll
      for (int u = 0; u < kUnroll; ++u)
        tm = fmaxf(tm, fmaxf(fmaxf(xs[u][0], xs[u][1]), fmaxf(xs[u][2], xs[u][3])));
      float ts = 0.f;
#pragma unroll
      for (int u = 0; u < kUnroll; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) ts += __builtin_amdgcn_exp2f((xs[u][e] - tm) * kLog2e);   // absent: exp(-inf) = 0
      merge_ms(m, s, tm, ts);
      if (trow) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          const int c = base + u * 4 * kThreads;
          if (c < c1v) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const bool gt = xt[u][e] > bv;
              bv = gt ? xt[u][e] : bv;
              bi = gt ? c + e : bi;
            }
          }
        }
      }
    }
    const int c = c1v + tid;               // the chunk's last (vocab % 4) elements
    if (c < c1) add_one(srow[c], c, trow ? trow[c] : 0.f);
  } else {
    for (int c = c0 + tid; c < c1; c += kThreads) add_one(srow[c], c, trow ? trow[c] : 0.f);
  }
  uint64_t key = bi >= 0 ? pack_key(bv, bi) : (first >= 0 ? pack_key(-INFINITY, first) : 0ull);

  // workgroup reduction of (m, s) and of the teacher key
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const float m2 = shfl_xor_f(m, o), s2 = shfl_xor_f(s, o);
    merge_ms(m, s, m2, s2);
    key = umax64(key, shfl_xor_u64(key, o));
  }
  if ((tid & 63) == 0) {
    red_m[tid >> 6] = m;
    red_s[tid >> 6] = s;
    red_k[tid >> 6] = key;
  }
  __syncthreads();
  uint32_t* row_counter = counter_line(p.counters, r);
  const __amdgpu_buffer_rsrc_t rec = make_rsrc(p.part + (int64_t)r * p.nsplit * 4, (uint32_t)(p.nsplit * 16));
  if (tid == 0) {
    for (int w = 1; w < kThreads / kWave; ++w) {
      merge_ms(m, s, red_m[w], red_s[w]);
      key = umax64(key, red_k[w]);
    }
    bool done = true;
    if (p.nsplit > 1) {
      store16_coherent(rec, (uint32_t)split * 16,
                       f32x4{m, s, __uint_as_float((uint32_t)key), __uint_as_float((uint32_t)(key >> 32))});
      wait_vmem();
      done = arrive(row_counter, (uint32_t)p.nsplit);
      if (done) reset_counter(row_counter);
    }
    if (done) {
      if (p.nsplit > 1) {             // merge the chunk records in chunk order
        m = -INFINITY;
        s = 0.f;
        key = 0ull;
        for (int c = 0; c < p.nsplit; ++c) {
          const f32x4 v = load16_coherent(rec, (uint32_t)c * 16);
          merge_ms(m, s, v[0], v[1]);
          key = umax64(key, ((uint64_t)__float_as_uint(v[3]) << 32) | __float_as_uint(v[2]));
        }
      }
      const int tgt = p.teacher ? (int)(0xFFFFFFFFu - (uint32_t)key) : p.targets[r];
      const float lse = m + __logf(s);
      const bool ok = tgt >= 0 && tgt < p.vocab;
      p.loss_out[r] = ok ? lse - srow[tgt] : __builtin_nanf("");
      if (p.target_out) p.target_out[r] = ok ? tgt : -1;
      if (p.lse_out) p.lse_out[r] = lse;
    }
  }
}

__global__ __launch_bounds__(kThreads) void sample_kernel(const float* u, int32_t count, SampleTable t, int32_t* out) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i >= count) return;
  const float x = u[i];
  int j = 0;
  while (j < t.n - 1 && !(x < t.thr[j])) ++j;
  out[i] = t.budgets[j];
}

}  // namespace

CePlan plan_ce(int rows, int vocab) {
  CePlan pl;
  int64_t want = ((int64_t)kTargetBlocks + rows - 1) / rows;
  const int64_t max_split = ((int64_t)vocab + 4 * kThreads - 1) / (4 * kThreads);
  const int64_t min_split = ((int64_t)vocab + 4 * kThreads * kUnroll - 1) / (4 * kThreads * kUnroll);
  if (want > max_split) want = max_split;
  if (want < min_split) want = min_split;
  if (want < 1) want = 1;
  int64_t chunk = ((int64_t)vocab + want - 1) / want;
  chunk = (chunk + 3) & ~int64_t(3);
  pl.chunk = (int)chunk;
  pl.nsplit = (int)((vocab + chunk - 1) / chunk);
  pl.record_bytes = pl.nsplit > 1 ? align256((size_t)rows * pl.nsplit * 16) : 0;
  pl.ws_bytes = BD_WS_COUNTER_BYTES + pl.record_bytes;
  return pl;
}

hipError_t launch_ce(const CeParams& p, hipStream_t stream) {
  hipLaunchKernelGGL(ce_kernel, dim3(p.rows * p.nsplit), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_sample(const float* u, int32_t count, const SampleTable& t, int32_t* out, hipStream_t stream) {
  const unsigned nb = (unsigned)(((int64_t)count + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(sample_kernel, dim3(nb), dim3(kThreads), 0, stream, u, count, t, out);
  return hipGetLastError();
}

}  // namespace bd
