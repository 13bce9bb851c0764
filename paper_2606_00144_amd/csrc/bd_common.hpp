// Device-side building blocks shared by the libbd kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bd.h"

namespace bd {

constexpr int kD = BD_HEAD_DIM;   // head dimension, fixed at 128
constexpr int kWave = 64;         // CDNA wavefront width
constexpr int kNumXcd = 8;        // MI355X: 256 CUs in 8 accelerator complex dies

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Device copy of bd_kv_desc (kernel argument).
struct KvView {
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* seq_lens;
  const int32_t* page_table;
  int64_t stride_seq, stride_head, stride_tok, stride_page;
  int32_t num_seqs, num_kv_heads, max_seq_len;
  int32_t page_size, max_pages_per_seq, num_pages;
};

inline KvView make_kv_view(const bd_kv_desc& d) {
  KvView v;
  v.k = d.k; v.v = d.v; v.seq_lens = d.seq_lens; v.page_table = d.page_table;
  v.stride_seq = d.stride_seq; v.stride_head = d.stride_head; v.stride_tok = d.stride_tok;
  v.stride_page = d.stride_page;
  v.num_seqs = d.num_seqs; v.num_kv_heads = d.num_kv_heads; v.max_seq_len = d.max_seq_len;
  v.page_size = d.page_size; v.max_pages_per_seq = d.max_pages_per_seq; v.num_pages = d.num_pages;
  return v;
}

// Cache length of sequence s, clamped to [0, max_seq_len].
__device__ inline int seq_len(const KvView& kv, int s) {
  int L = kv.seq_lens[s];
  return L < 0 ? 0 : (L > kv.max_seq_len ? kv.max_seq_len : L);
}

// Element offset of row t of KV head g of sequence s, or -1 when the row's
// page number is outside the pool (the key is then treated as absent).
template <bool PAGED>
__device__ inline int64_t row_offset(const KvView& kv, int s, int g, int t) {
  if constexpr (PAGED) {
    const int pg = kv.page_table[(int64_t)s * kv.max_pages_per_seq + t / kv.page_size];
    if ((unsigned)pg >= (unsigned)kv.num_pages) return -1;
    return (int64_t)pg * kv.stride_page + (int64_t)g * kv.stride_head + (int64_t)(t % kv.page_size) * kv.stride_tok;
  } else {
    return (int64_t)s * kv.stride_seq + (int64_t)g * kv.stride_head + (int64_t)t * kv.stride_tok;
  }
}

// Workgroups are handed to the 8 XCDs round-robin (block b runs on XCD b % 8).
// Remap so that each XCD receives one contiguous range of logical ids: work
// items that share data (the splits of one (sequence, head) unit, the row
// blocks of one key range) then share one XCD's L2.
__device__ inline int xcd_remap(int b, int n) {
  const int q = n / kNumXcd, r = n % kNumXcd;
  const int x = b % kNumXcd, j = b / kNumXcd;
  return x * q + (x < r ? x : r) + j;
}

// n / d for 0 <= n < 2^22, d >= 1, with inv_d = 1/d to within an ulp: the float estimate is within
// one of the quotient, and one correction each way makes it exact (a VALU integer division costs
// tens of instructions).
__device__ inline int div_small(int n, int d, float inv_d) {
  int q = (int)((float)n * inv_d);
  q += (q + 1) * d <= n ? 1 : 0;
  q -= q * d > n ? 1 : 0;
  return q;
}
__device__ inline int div_small(int n, int d) { return div_small(n, d, __builtin_amdgcn_rcpf((float)d)); }

// ---- cross-lane reductions ------------------------------------------------

// xor-shuffle through the LDS crossbar (ds_bpermute); works across all 64 lanes.
__device__ inline float shfl_xor_f(float x, int m) {
  const int src = (int)(threadIdx.x ^ m) & (kWave - 1);
  return __int_as_float(__builtin_amdgcn_ds_bpermute(src << 2, __float_as_int(x)));
}

// Reductions over lane pairs (l, l^16) and (l, l^32) with the gfx950 row-swap
// instructions: VALU only, no LDS crossbar.
__device__ inline float max_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float sum_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ inline float sum_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// ---- LDS reads the compiler does not see ----------------------------------
//
// While direct-to-LDS loads are in flight the compiler's wait analysis makes
// every LDS read wait for all of them (vmcnt(0)).  The streaming loop
// therefore reads LDS with inline asm that issues its loads AND waits for them
// (lgkmcnt(0)) in one statement: the compiler only sees the results once they
// have landed, so no use can be scheduled early.
__device__ inline uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// Sum over each aligned group of 16 lanes, result in every lane (DPP only).
__device__ inline float sum16(float x) {
  x += __builtin_amdgcn_update_dpp(0.0f, x, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
  x += __builtin_amdgcn_update_dpp(0.0f, x, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
  x += __builtin_amdgcn_update_dpp(0.0f, x, 0x141, 0xF, 0xF, false);  // row_half_mirror
  x += __builtin_amdgcn_update_dpp(0.0f, x, 0x140, 0xF, 0xF, false);  // row_mirror
  return x;
}

// ---- data handed from one workgroup to another -----------------------------
//
// The splits of a unit publish partial results for the last workgroup to
// finish.  They are written and read with relaxed agent-scope atomic accesses,
// which gfx950 performs at the device coherence point (the `sc1` cache
// policy), so neither side needs a cache-wide fence: the writer waits until
// its stores are acknowledged (vmcnt(0)) before bumping the counter, and the
// reader issues its loads only after seeing the final count.  (A
// __threadfence() here would write back and invalidate the whole L2 of the
// XCD once per workgroup.)
__device__ inline void store_coherent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void store_coherent(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline float load_coherent(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline uint64_t load_coherent(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// 16-byte coherent accesses (buffer_store/load_dwordx4 with the sc1 policy) through a buffer
// resource over [base, base + bytes); accesses outside the range are dropped (stores) or read 0.
constexpr int kPolicySc1 = 16;
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}
__device__ inline void store16_coherent(__amdgpu_buffer_rsrc_t r, uint32_t off, f32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, (int)off, 0, kPolicySc1);
}
__device__ inline f32x4 load16_coherent(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kPolicySc1));
}
// Wait until every vector memory operation of this wave has completed.
__device__ inline void wait_vmem() {
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0), expcnt/lgkmcnt unconstrained
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}
// Count one finished split of a unit; true in the workgroup that finished last.
__device__ inline bool arrive(uint32_t* counter, uint32_t total) {
  const uint32_t prev = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  return prev == total - 1;
}
__device__ inline void reset_counter(uint32_t* counter) {
  __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Line i of the workspace's counter region.
__device__ inline uint32_t* counter_line(uint32_t* region, int64_t i) {
  return region + i * (BD_WS_COUNTER_STRIDE / 4);
}
__device__ inline void atomic_max_coherent(uint64_t* p, uint64_t v) {
  __hip_atomic_fetch_max(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---- bf16 helpers ---------------------------------------------------------

__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Two floats -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ inline bf16x8 as_bf16x8(u32x4 w) { return __builtin_bit_cast(bf16x8, w); }

__device__ inline u32x4 load16(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }

// Order-preserving map of a finite float to uint32 (-0.0 folds onto +0.0).
__device__ inline uint32_t float_order_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

}  // namespace bd
