// TopB eviction with a protected recent window and in-place compaction
// (Eq. (1), first two lines), one workgroup per (sequence, layer, KV head).
//
// Selection: of the candidate slots [0, n-W) keep the B-W with the largest
// score, ties to the lower slot. Scores are compared through an order-
// preserving map of their float32 bit patterns (32-bit keys), so the order
// (key desc, slot asc) is strict and exactly B-W slots are kept even for
// unusual inputs. One wavefront finds the threshold key T, the (B-W)-th
// largest, by a bitwise radix select from the most significant bit: at each
// bit it counts (ballot + popcount) the candidates that match T's bits
// decided so far and have this bit set; if they are at least the number still
// wanted the bit of T is 1, else they are all kept and the count wanted drops
// by theirs. That is 32 ballot rounds over n-W keys (held in registers up to
// 256 candidates), O(n) work where counting every candidate's rank against
// all others is O(n^2). The kept slots are then the keys above T and the
// lowest-slot keys equal to T, and their destinations a ballot prefix count
// in slot order. The window [n-W, n) is always kept.
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

// Order-preserving 32-bit key of a float32 score; -0 and +0 map to one key
// (they compare equal, so their tie goes to the lower slot).
__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

constexpr int kThreads = 256;
constexpr int kRegKeys = 4;  // candidate keys per lane held in registers by the select (n - W <= 256)
constexpr int kItems = 1;  // 16-byte items per thread per tensor per chunk

__global__ __launch_bounds__(kThreads) void evict_topb_kernel(EvictParams p, int row_units) {
  extern __shared__ uint32_t lds[];
  const int unit = blockIdx.x;  // ((s * L) + l) * Hkv + h
  const int s = unit / (p.L * p.Hkv);
  int n = p.len[s];
  if (p.len_out && unit % (p.L * p.Hkv) == 0 && threadIdx.x == 0)
    p.len_out[s] = n > p.B + p.buffer ? p.B : n;
  if (n <= p.B + p.buffer) return;
  if (n > p.cap) n = p.cap;
  const int tid = threadIdx.x;
  const int nc = n - p.W;
  const int take = p.B - p.W;

  uint32_t *key = lds;                                    // [cap]
  int *kept = reinterpret_cast<int *>(lds + p.cap);       // [B]
  __shared__ int first_moved;

  const float *sc = p.scores + (size_t)unit * p.cap;
  for (int j = tid; j < nc; j += kThreads) key[j] = order_key(sc[j]);
  if (tid == 0) first_moved = p.B;
  __syncthreads();

  if (tid < kWave) {
    // Candidate j = 64 r + lane; keys past nc are never counted.
    const int lane = tid;
    const uint64_t below = (1ull << lane) - 1ull;
    const bool inreg = nc <= kWave * kRegKeys;
    uint32_t kr[kRegKeys];
#pragma unroll
    for (int r = 0; r < kRegKeys; r++) kr[r] = (inreg && kWave * r + lane < nc) ? key[kWave * r + lane] : 0u;
    uint32_t T = 0u;
    int need = take;  // >= 1: nc >= B > B - W
    for (int bit = 31; bit >= 0; bit--) {
      const uint32_t hi = ~((2u << bit) - 1u);  // the bits of T decided so far (none at bit 31)
      const uint32_t want = T & hi;
      int c = 0;
      if (inreg) {
#pragma unroll
        for (int r = 0; r < kRegKeys; r++)
          c += __popcll(__ballot(kWave * r + lane < nc && (kr[r] & hi) == want && ((kr[r] >> bit) & 1u)));
      } else {
        for (int j0 = 0; j0 < nc; j0 += kWave) {
          const int j = j0 + lane;
          const uint32_t k = j < nc ? key[j] : 0u;
          c += __popcll(__ballot(j < nc && (k & hi) == want && ((k >> bit) & 1u)));
        }
      }
      if (c >= need) T |= 1u << bit;
      else need -= c;
    }
    // Keep every key above T and the `need` lowest-slot keys equal to T, in
    // slot order: destination = kept candidates before this one.
    int base = 0, eq_seen = 0;
    for (int j0 = 0; j0 < nc; j0 += kWave) {
      const int j = j0 + lane;
      const uint32_t k = j < nc ? (inreg ? kr[0] : key[j]) : 0u;
      const bool eq = j < nc && k == T;
      const uint64_t eqm = __ballot(eq);
      const bool keep = j < nc && (k > T || (eq && eq_seen + __popcll(eqm & below) < need));
      const uint64_t km = __ballot(keep);
      if (keep) kept[base + __popcll(km & below)] = j;
      base += __popcll(km);
      eq_seen += __popcll(eqm);
      if (inreg) {
#pragma unroll
        for (int r = 0; r + 1 < kRegKeys; r++) kr[r] = kr[r + 1];
      }
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
  const size_t lds = (size_t)(p.cap + p.B) * sizeof(uint32_t);
  hipLaunchKernelGGL(evict_topb_kernel, dim3(p.S * p.L * p.Hkv), dim3(kThreads), lds, stream, p,
                     row_units);
  return hipGetLastError();
}

}  // namespace kvr
