// Per-round cache updates (Alg. 2: the caches are updated with the appended tokens).
//
// Appending writes the new rows' K and V at positions L_s .. L_s+n-1 and, for
// the drafter's sparse cache, appends those positions to every KV head's index
// list, then advances the lengths (every row copy reads the old length first).
// Up to kFusedRows rows one workgroup per sequence does both, the advance after
// a barrier, in one launch: the round's appends are single rows (the drafts) and
// gamma+1 rows (the verifier), and a second launch of a few microseconds'
// latency per append cost more than the copies.  Longer appends take one
// workgroup per (sequence, row) and a second launch for the lengths (stream
// order separates the two).  Rollback keeps the accepted speculative rows after
// verification.  All of it is integer and byte work: one 16-byte load and store
// per lane per row chunk.

#include "bd_common.hpp"
#include "bd_kernels.hpp"

namespace bd {
namespace {

constexpr int kThreads = 256;
constexpr int kChunks = kD * 2 / 16;   // 16-byte chunks of a 128-element bf16 row
constexpr int kFusedRows = 16;         // appends of up to this many rows take the one-launch kernel

__device__ inline int clamp_len(int L, int cap) { return L < 0 ? 0 : (L > cap ? cap : L); }

// Element offset of cache row t of sequence s (head 0), or -1 when its page is outside the pool.
__device__ inline int64_t row_base(const KvView& kv, int s, int t) {
  if (kv.page_table) {
    const int pg = kv.page_table[(int64_t)s * kv.max_pages_per_seq + t / kv.page_size];
    return (unsigned)pg < (unsigned)kv.num_pages ? (int64_t)pg * kv.stride_page + (int64_t)(t % kv.page_size) * kv.stride_tok
                                                 : -1;
  }
  return (int64_t)s * kv.stride_seq + (int64_t)t * kv.stride_tok;
}

// Chunk r of head g of new row i of sequence s (K chunks then V chunks) to the cache row at base.
__device__ inline void copy_chunk(const AppendParams& p, int s, int i, int g, int r, int64_t base) {
  const bool is_v = r >= kChunks;
  const int c = is_v ? r - kChunks : r;
  const int64_t src = (((int64_t)s * p.n + i) * p.kv.num_kv_heads + g) * kD + 8 * c;
  const int64_t dst = base + (int64_t)g * p.kv.stride_head + 8 * c;
  uint16_t* cache = const_cast<uint16_t*>(is_v ? p.kv.v : p.kv.k);
  *reinterpret_cast<u32x4*>(cache + dst) = load16((is_v ? p.v_new : p.k_new) + src);
}

// Advance sequence s's length (and sparse count) by the rows an append of p.n rows wrote.
__device__ inline void advance(const AppendParams& p, int s, int L) {
  const int cap = p.kv.max_seq_len;
  const int w = p.n < cap - L ? p.n : cap - L;
  const_cast<int32_t*>(p.kv.seq_lens)[s] = L + w;
  if (p.idx) {
    int m = p.nsel[s];
    m = m < 0 ? 0 : (m > p.ld_idx ? p.ld_idx : m);
    const int a = w < p.ld_idx - m ? w : p.ld_idx - m;
    p.nsel[s] = m + a;
  }
}

// Block s: every new row of sequence s (n <= kFusedRows), then its length.  All reads of the old
// length and count happen before the barrier; thread 0 writes the new ones after it.
__global__ __launch_bounds__(kThreads) void append_fused_kernel(AppendParams p) {
  const int s = blockIdx.x;
  const int cap = p.kv.max_seq_len;
  const int L = clamp_len(p.kv.seq_lens[s], cap);
  int m = 0;
  if (p.idx) {
    m = p.nsel[s];
    m = m < 0 ? 0 : (m > p.ld_idx ? p.ld_idx : m);
  }
  const int per_head = 2 * kChunks;                       // K chunks then V chunks
  const int per_row = p.kv.num_kv_heads * per_head;
  for (int w = threadIdx.x; w < p.n * per_row; w += kThreads) {
    const int i = w / per_row, r0 = w - i * per_row;
    const int t = L + i;
    if (t >= cap) continue;                                 // past the capacity: dropped
    const int64_t base = row_base(p.kv, s, t);
    if (base >= 0) copy_chunk(p, s, i, r0 / per_head, r0 % per_head, base);
  }
  if (p.idx)
    for (int w = threadIdx.x; w < p.n * p.kv.num_kv_heads; w += kThreads) {
      const int i = w / p.kv.num_kv_heads, g = w - i * p.kv.num_kv_heads;
      if (L + i < cap && m + i < p.ld_idx) p.idx[((int64_t)s * p.kv.num_kv_heads + g) * p.ld_idx + m + i] = L + i;
    }
  __syncthreads();
  if (threadIdx.x == 0) advance(p, s, L);
}

// Block (s, i): new row i of sequence s, every KV head; thread -> (head, K or V, chunk).
__global__ __launch_bounds__(kThreads) void append_rows_kernel(AppendParams p) {
  const int s = blockIdx.x / p.n, i = blockIdx.x % p.n;
  const int cap = p.kv.max_seq_len;
  const int L = clamp_len(p.kv.seq_lens[s], cap);
  const int t = L + i;
  if (t >= cap) return;                                   // past the capacity: dropped
  const int64_t base = row_base(p.kv, s, t);
  const int per_head = 2 * kChunks;                       // K chunks then V chunks
  if (base >= 0)
    for (int w = threadIdx.x; w < p.kv.num_kv_heads * per_head; w += kThreads) copy_chunk(p, s, i, w / per_head, w % per_head, base);
  if (p.idx) {
    int m = p.nsel[s];
    m = m < 0 ? 0 : (m > p.ld_idx ? p.ld_idx : m);
    if (m + i < p.ld_idx)
      for (int g = threadIdx.x; g < p.kv.num_kv_heads; g += kThreads)
        p.idx[((int64_t)s * p.kv.num_kv_heads + g) * p.ld_idx + m + i] = t;
  }
}

// Thread s: advance the length (and the sparse count) by what append_rows_kernel wrote.
__global__ __launch_bounds__(kThreads) void append_advance_kernel(AppendParams p) {
  const int s = blockIdx.x * kThreads + threadIdx.x;
  if (s >= p.kv.num_seqs) return;
  advance(p, s, clamp_len(p.kv.seq_lens[s], p.kv.max_seq_len));
}

// Thread s: keep the accepted prefix of the speculative rows.  With the lengths from before the
// speculative appends, a count becomes min(count, base + accepted) (rows an append dropped were never
// counted); without them, spec - accepted is subtracted.
__global__ __launch_bounds__(kThreads) void rollback_kernel(RollbackParams p) {
  const int s = blockIdx.x * kThreads + threadIdx.x;
  if (s >= p.S) return;
  int a = p.accept[s];
  a = a < 0 ? 0 : (a > p.spec ? p.spec : a);
  auto keep = [&](int cur, const int32_t* base) {
    const int64_t v = base ? (int64_t)base[s] + a : (int64_t)cur - (p.spec - a);
    const int64_t c = v < cur ? v : cur;
    return (int)(c < 0 ? 0 : c);
  };
  p.seq_lens[s] = keep(p.seq_lens[s], p.base_lens);
  if (p.nsel) p.nsel[s] = keep(p.nsel[s], p.base_nsel);
}

}  // namespace

hipError_t launch_append(const AppendParams& p, hipStream_t stream) {
  if (p.n <= kFusedRows) {
    hipLaunchKernelGGL(append_fused_kernel, dim3(p.kv.num_seqs), dim3(kThreads), 0, stream, p);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(append_rows_kernel, dim3(p.kv.num_seqs * p.n), dim3(kThreads), 0, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const unsigned nb = (unsigned)(((int64_t)p.kv.num_seqs + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(append_advance_kernel, dim3(nb), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_rollback(const RollbackParams& p, hipStream_t stream) {
  const unsigned nb = (unsigned)(((int64_t)p.S + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(rollback_kernel, dim3(nb), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace bd
