// Data movement around the decode loop: forking candidates from a trajectory
// state (or retaining a candidate as the state) and appending a step's tokens
// in bulk (App. C, the fork-based engine; Alg. 1, retain / append-and-evict).
//
// Both are plain HBM copies of contiguous slot ranges: in the [cap][D] layout
// of each (sequence, layer, KV head) the live slots [0, n) of K and of V are
// one contiguous run of n * D elements, and an append writes one contiguous
// run of T * D elements. Workgroups stream 16-byte vectors with all of a
// round's loads issued before its stores, which are non-temporal.
//
// Fork: one workgroup per (group of kGroup consecutive destinations, layer,
// KV head, K or V, chunk of kChunkRounds rounds of slots). Within a group,
// destinations that share a source form runs; each round loads a piece of the
// run's source once and stores it to every destination of the run. Forking N
// candidates from one state (destinations s*N .. s*N+N-1 reading source s)
// therefore reads each source byte from HBM once, whatever the L2 does, and
// the stores stream at full rate.
#include <hip/hip_runtime.h>

#include "kvr_device.h"
#include "kvr_internal.h"

namespace kvr {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

constexpr int kGroup = 8;
// Fork workgroup shape: vectors per thread per round, rounds per workgroup,
// and whether K and V go to workgroups of their own. On the 7B fork shape
// (16 states x 8 candidates, 640 slots) one round of 2 vectors with K and V
// apart (26 VGPRs, 8 waves per SIMD) measured 991 us, against 1009 us for 4
// vectors with K and V together (119 VGPRs, 4 waves), 998 us for 2 together,
// 1607-1729 us for 8 (one wave per SIMD), and 1101 us for whole runs per
// workgroup dispatched group-fastest. Looping workgroups over the same items
// (a grid of 1-4 times the resident count) measured 1283-1458 us: each
// workgroup's items then run one after another, where the dispatcher
// overlaps many small workgroups.
constexpr int kForkUnroll = 2;
constexpr int kChunkRounds = 1;
constexpr bool kSplitKV = true;
static_assert(kForkMaxLH * (kSplitKV ? 2 : 1) <= 65535 && kForkMaxDst / kGroup <= 65535,
              "fork limits exceed the grid's y and z dimensions");

// Loads one round (U vectors per thread) of a run's source rows.
template <int U>
__device__ __forceinline__ void load_round(const u32x4 *__restrict__ src, int base, int nv, u32x4 (&r)[U]) {
#pragma unroll
  for (int a = 0; a < U; a++) {
    const int i = base + a * kThreads;
    if (i < nv) r[a] = src[i];
  }
}

// Non-temporal stores: the copies are not read again by this kernel, and
// measured 4-5% faster than ordinary stores for the fork's write stream.
template <int U>
__device__ __forceinline__ void store_round(u32x4 *__restrict__ dst, int base, int nv, const u32x4 (&r)[U]) {
#pragma unroll
  for (int a = 0; a < U; a++) {
    const int i = base + a * kThreads;
    if (i < nv) __builtin_nontemporal_store(r[a], dst + i);
  }
}

// grid (chunks, L * Hkv (x 2 with kSplitKV), destination groups). Workgroups
// are dispatched chunk-fastest and group-slowest, so the ones resident at any
// moment write adjacent pieces of the same few destination caches: 1009
// against 1097 us on the 7B fork shape with the same workgroups dispatched
// group-fastest (which spreads the resident writes over every destination).
__global__ __launch_bounds__(kThreads) void fork_kernel(ForkParams p, int row_units) {
  constexpr int kRound = kForkUnroll * kThreads;
  // This workgroup's vectors [v0, v1) of every run: whole rounds, so the
  // rounds of adjacent chunks do not overlap.
  const int v0 = blockIdx.x * kChunkRounds * kRound, v1 = v0 + kChunkRounds * kRound;
  const int kv = kSplitKV ? (int)(blockIdx.y & 1) : 0;  // 0: K (and V unless split), 1: V
  const int lh = kSplitKV ? (int)(blockIdx.y >> 1) : (int)blockIdx.y;  // l * Hkv + h
  const int s0 = blockIdx.z * kGroup;
  const int tid = threadIdx.x;
  const int cmax = p.cap_src < p.cap_dst ? p.cap_src : p.cap_dst;
  // Per destination of the group: source row (-1: skip) and slots to copy.
  int src[kGroup], nn[kGroup];
  int nvmax = 0;
#pragma unroll
  for (int j = 0; j < kGroup; j++) {
    const int s = s0 + j;
    int r = -1, n = 0;
    if (s < p.S_dst) {
      r = p.src_index[s];
      n = p.len[s];
      n = n < 0 ? 0 : (n > cmax ? cmax : n);
      if (r < 0 || r >= p.S_src || (p.same && r == s) || n == 0) r = -1;
    }
    src[j] = r;
    nn[j] = r < 0 ? 0 : n;
    nvmax = max(nvmax, nn[j] * row_units);
  }
  nvmax = min(nvmax, v1);
  const size_t row_vec = (size_t)row_units;
  const size_t sstride = (size_t)p.L * p.Hkv;
  const u32x4 *sk = static_cast<const u32x4 *>(kv ? p.sv : p.sk);
  const u32x4 *sv = static_cast<const u32x4 *>(p.sv);
  u32x4 *dk = static_cast<u32x4 *>(kv ? p.dv : p.dk);
  u32x4 *dv = static_cast<u32x4 *>(p.dv);
  for (int base = v0 + tid; base < nvmax; base += kRound) {
    int j = 0;
    while (j < kGroup) {
      const int r = src[j];
      if (r < 0) {
        j++;
        continue;
      }
      // Run j .. e-1 shares source r; read as far as its longest member.
      int e = j + 1, nvr = nn[j] * row_units;
      while (e < kGroup && src[e] == r) {
        nvr = max(nvr, nn[e] * row_units);
        e++;
      }
      const size_t so = ((size_t)r * sstride + lh) * p.cap_src * row_vec;
      u32x4 rk[kForkUnroll], rv[kForkUnroll];
      load_round(sk + so, base, nvr, rk);
      if (!kSplitKV) load_round(sv + so, base, nvr, rv);
      for (int k = j; k < e; k++) {
        const size_t d = ((size_t)(s0 + k) * sstride + lh) * p.cap_dst * row_vec;
        store_round(dk + d, base, nn[k] * row_units, rk);
        if (!kSplitKV) store_round(dv + d, base, nn[k] * row_units, rv);
      }
      j = e;
    }
  }
  if ((p.dpos || p.dsc) && kv == 0) {
    // The slots of this chunk: [v0, v1) / row_units, a partition of the run.
    const int t0 = v0 / row_units, t1 = v1 / row_units;
#pragma unroll
    for (int j = 0; j < kGroup; j++) {
      if (src[j] < 0) continue;
      const size_t su = (size_t)src[j] * sstride + lh;
      const size_t du = (size_t)(s0 + j) * sstride + lh;
      const int te = nn[j] < t1 ? nn[j] : t1;
      for (int t = t0 + tid; t < te; t += kThreads) {
        if (p.dpos) p.dpos[du * p.cap_dst + t] = p.spos[su * p.cap_src + t];
        if (p.dsc) p.dsc[du * p.cap_dst + t] = p.ssc[su * p.cap_src + t];
      }
    }
  }
}

// grid (units, chunks): chunk c of unit u copies vectors
// [c * kUnroll * kThreads, (c + 1) * kUnroll * kThreads) of the unit's T rows.
__global__ __launch_bounds__(kThreads) void append_kernel(AppendParams p, int row_units) {
  const int unit = blockIdx.x;  // (s * L + l) * Hkv + h
  const int s = unit / (p.L * p.Hkv);
  int n = p.len[s];
  n = n < 0 ? 0 : (n > p.cap ? p.cap : n);
  const int rows = p.T < p.cap - n ? p.T : p.cap - n;  // rows that fit
  const int nv = rows * row_units;
  const int v0 = blockIdx.y * kUnroll * kThreads;
  const int tid = threadIdx.x;
  const size_t row_vec = (size_t)row_units;
  const u32x4 *sk = static_cast<const u32x4 *>(p.k_new) + (size_t)unit * p.T * row_vec;
  const u32x4 *sv = static_cast<const u32x4 *>(p.v_new) + (size_t)unit * p.T * row_vec;
  u32x4 *dk = static_cast<u32x4 *>(p.k) + ((size_t)unit * p.cap + n) * row_vec;
  u32x4 *dv = static_cast<u32x4 *>(p.v) + ((size_t)unit * p.cap + n) * row_vec;
  u32x4 rk[kUnroll], rv[kUnroll];
#pragma unroll
  for (int a = 0; a < kUnroll; a++) {
    const int i = v0 + tid + a * kThreads;
    if (i < nv) {
      rk[a] = sk[i];
      rv[a] = sv[i];
    }
  }
#pragma unroll
  for (int a = 0; a < kUnroll; a++) {
    const int i = v0 + tid + a * kThreads;
    if (i < nv) {  // non-temporal, as the fork's (measured 9% faster here)
      __builtin_nontemporal_store(rk[a], dk + i);
      __builtin_nontemporal_store(rv[a], dv + i);
    }
  }
  if (p.pos_new && blockIdx.y == 0) {
    int32_t *dp = p.pos + (size_t)unit * p.cap + n;
    const int32_t *sp = p.pos_new + (size_t)s * p.T;
    for (int j = tid; j < rows; j += kThreads) dp[j] = sp[j];
  }
}

}  // namespace

hipError_t launch_fork(const ForkParams &p, hipStream_t stream) {
  const int row_units = p.D * p.esz / 16;
  // Chunks cover the longest run a destination can have (its cache's or the
  // source's capacity); those past a run's live length return at once.
  const long cmax = p.cap_src < p.cap_dst ? p.cap_src : p.cap_dst;
  const long chunk_vec = (long)kChunkRounds * kForkUnroll * kThreads;
  const int chunks = (int)((cmax * row_units + chunk_vec - 1) / chunk_vec);
  const dim3 grid(chunks > 0 ? chunks : 1, p.L * p.Hkv * (kSplitKV ? 2 : 1), (p.S_dst + kGroup - 1) / kGroup);
  hipLaunchKernelGGL(fork_kernel, grid, dim3(kThreads), 0, stream, p, row_units);
  return hipGetLastError();
}

hipError_t launch_append(const AppendParams &p, hipStream_t stream) {
  const int row_units = p.D * p.esz / 16;
  const long nv = (long)p.T * row_units;
  const int chunks = (int)((nv + kUnroll * kThreads - 1) / (kUnroll * kThreads));
  hipLaunchKernelGGL(append_kernel, dim3(p.S * p.L * p.Hkv, chunks), dim3(kThreads), 0, stream, p,
                     row_units);
  return hipGetLastError();
}

}  // namespace kvr
