// TopB eviction with a protected recent window and in-place compaction
// (Eq. (1), first two lines), one workgroup per (sequence, layer, KV head).
//
// Selection: of the candidate slots [0, n-W) keep the B-W with the largest
// score, ties to the lower slot. Each candidate's rank under the strict total
// order (score desc, slot asc) is counted directly against all others held in
// LDS; rank < B-W means kept. Scores are compared through an order-preserving
// map of their float32 bit patterns, so the ranks form a permutation and
// exactly B-W slots are kept even for unusual inputs. The window [n-W, n) is
// always kept.
//
// Compaction: kept slot k_i moves to slot i. Since k_i >= i, destinations are
// processed in ascending chunks of one 16-byte item of K and one of V per
// thread (16 rows of bf16 D = 128): all sources of a chunk are read into
// registers, the reads are waited for, the workgroup synchronises, then the
// chunk is written. A chunk's writes land on rows below every later chunk's
// sources, so nothing is overwritten before it is read. Rows already in place
// (the kept prefix before the first evicted slot) are not touched. Larger
// chunks (up to 128 rows per read phase) measured slower: the registers they
// hold cut the number of heads in flight, which is what hides the latency.
#include <hip/hip_runtime.h>

#include "kvr_device.h"
#include "kvr_internal.h"

namespace kvr {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t order_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

constexpr int kThreads = 256;
constexpr int kItems = 1;  // 16-byte items per thread per tensor per chunk

__global__ __launch_bounds__(kThreads) void evict_topb_kernel(EvictParams p, int row_units) {
  extern __shared__ uint32_t lds[];
  const int unit = blockIdx.x;  // ((s * L) + l) * Hkv + h
  const int s = unit / (p.L * p.Hkv);
  int n = p.len[s];
  if (n <= p.B + p.buffer) return;
  if (n > p.cap) n = p.cap;
  const int tid = threadIdx.x;
  const int nc = n - p.W;
  const int take = p.B - p.W;

  uint32_t *key = lds;                                    // [cap]
  int *flag = reinterpret_cast<int *>(lds + p.cap);       // [cap]
  int *kept = reinterpret_cast<int *>(lds + 2 * p.cap);   // [B]
  __shared__ int first_moved;

  const float *sc = p.scores + (size_t)unit * p.cap;
  for (int j = tid; j < nc; j += kThreads) key[j] = order_key(sc[j]);
  if (tid == 0) first_moved = p.B;
  __syncthreads();

  for (int j = tid; j < nc; j += kThreads) {
    const uint32_t kj = key[j];
    int rank = 0;
    for (int i = 0; i < nc; i++) {
      const uint32_t ki = key[i];
      rank += (ki > kj) | ((ki == kj) & (i < j));
    }
    flag[j] = rank < take;
  }
  __syncthreads();
  for (int j = tid; j < nc; j += kThreads) {
    if (flag[j]) {
      int dst = 0;
      for (int i = 0; i < j; i++) dst += flag[i];
      kept[dst] = j;
    }
  }
  for (int w = tid; w < p.W; w += kThreads) kept[take + w] = nc + w;
  __syncthreads();

  if (p.kept) {
    int32_t *ko = p.kept + (size_t)unit * p.B;
    for (int i = tid; i < p.B; i += kThreads) ko[i] = kept[i];
  }
  for (int i = tid; i < p.B; i += kThreads)
    if (kept[i] != i) atomicMin(&first_moved, i);
  __syncthreads();

  const size_t row_bytes = (size_t)row_units * 16;
  char *Kb = static_cast<char *>(p.k) + (size_t)unit * p.cap * row_bytes;
  char *Vb = static_cast<char *>(p.v) + (size_t)unit * p.cap * row_bytes;
  int32_t *pos = p.pos ? p.pos + (size_t)unit * p.cap : nullptr;
  const int chunk_rows = kThreads * kItems / row_units;  // <= kThreads (row_units >= 8)
  // first_moved is uniform; start at the chunk holding it.
  for (int c0 = first_moved; c0 < p.B; c0 += chunk_rows) {
    u32x4 kr[kItems], vr[kItems];
    int32_t pr = 0;
#pragma unroll
    for (int a = 0; a < kItems; a++) {
      const int e = tid + a * kThreads;  // item of the chunk: row e / row_units, 16 bytes e % row_units
      const int i = c0 + e / row_units;
      if (i < p.B) {
        const int src = kept[i];
        const int u = e % row_units;
        kr[a] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(Kb + (size_t)src * row_bytes) + u);
        vr[a] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(Vb + (size_t)src * row_bytes) + u);
      }
    }
    if (pos && tid < chunk_rows && c0 + tid < p.B) pr = pos[kept[c0 + tid]];
    // Every read of the chunk is performed before any thread writes.
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
#pragma unroll
    for (int a = 0; a < kItems; a++) {
      const int e = tid + a * kThreads;
      const int i = c0 + e / row_units;
      if (i < p.B) {
        const int u = e % row_units;
        // Non-temporal: the compacted rows are next read a decode step later.
        __builtin_nontemporal_store(kr[a], reinterpret_cast<u32x4 *>(Kb + (size_t)i * row_bytes) + u);
        __builtin_nontemporal_store(vr[a], reinterpret_cast<u32x4 *>(Vb + (size_t)i * row_bytes) + u);
      }
    }
    if (pos && tid < chunk_rows && c0 + tid < p.B) pos[c0 + tid] = pr;
    // Later chunks read only rows above this chunk's destinations, so they
    // need no wait for these writes.
  }
}

}  // namespace

hipError_t launch_evict_topb(const EvictParams &p, hipStream_t stream) {
  const int esz = p.dtype == 0 ? 4 : 2;
  const int row_units = p.D * esz / 16;
  const size_t lds = (size_t)(2 * p.cap + p.B) * sizeof(uint32_t);
  hipLaunchKernelGGL(evict_topb_kernel, dim3(p.S * p.L * p.Hkv), dim3(kThreads), lds, stream, p,
                     row_units);
  return hipGetLastError();
}

}  // namespace kvr
