// Device-side pieces of the token sampler fused with the entropy pass
// (Sec. 4.1 decoding setup: temperature, top-k, top-p): the per-wave
// candidate buffers of the k largest logits, the threshold selection by
// ballot counts, the Philox4x64-10 generator and the draw from the sorted
// candidates. Shared by the entropy kernels and the base-attention launch
// that samples the step's tokens alongside.
#pragma once

#include <hip/hip_runtime.h>

#include "entropy_common.h"

namespace kvr {
namespace {

// ---------------------------------------------------------------- sampler

__device__ __forceinline__ uint32_t order_bits(float x) {
  const uint32_t u = x == 0.f ? 0u : __float_as_uint(x);  // -0 ranks as +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float from_order_bits(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}
// Larger key = larger logit, then lower id. Every real key is > 0.
__device__ __forceinline__ uint64_t cand_key(float x, uint32_t id) {
  return ((uint64_t)order_bits(x) << 32) | (uint64_t)(~id);
}

constexpr int kKeep = 128;                        // entries kept by a compaction, at most
constexpr int kCandCap = kKeep + kWave;           // wave buffer: one offer adds <= 64
constexpr int kCandPerLane = kCandCap / kWave;    // 3

// Wave-wide count of entries >= t (entries are keys, 0 = empty; t >= 1).
template <int NPL>
__device__ __forceinline__ int wave_count_ge(const uint64_t (&v)[NPL], uint64_t t) {
  int c = 0;
#pragma unroll
  for (int i = 0; i < NPL; i++) c += __popcll(__ballot(v[i] >= t));
  return c;
}

// A threshold t with k <= count(entries >= t) <= cap, built bit by bit from
// the top with ballot counts only and stopped as soon as the count fits (with
// cap = k: exactly the k largest keys, as keys are unique). Returns 1 when
// all entries already fit.
template <int NPL>
__device__ __forceinline__ uint64_t select_threshold(const uint64_t (&v)[NPL], int k, int cap) {
  if (wave_count_ge(v, 1) <= cap) return 1;
  uint64_t t = 0;
  for (int b = 63; b >= 0; b--) {
    const uint64_t c = t | (1ull << b);
    const int n = wave_count_ge(v, c);
    if (n >= k) {
      t = c;
      if (n <= cap) break;
    }
  }
  return t;
}

// Stores the wave's keys >= t to out[0 ..) (unordered); returns how many.
template <int NPL>
__device__ __forceinline__ int wave_store_ge(uint64_t *out, const uint64_t (&v)[NPL], uint64_t t, int lane) {
  const uint64_t below = (1ull << lane) - 1ull;
  int base = 0;
#pragma unroll
  for (int i = 0; i < NPL; i++) {
    const bool m = v[i] >= t;
    const uint64_t b = __ballot(m);
    if (m) out[base + __popcll(b & below)] = v[i];
    base += __popcll(b);
  }
  return base;
}

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// A wave's candidate buffer: keys >= kmin are kept; logits below vmin cannot
// reach kmin (vmin is the logit part of kmin).
struct Cands {
  uint64_t *buf;
  int cnt;
  uint64_t kmin;
  float vmin;
};

// Keeps between k and cap of the buffered keys (cap = k: exactly the k best),
// unordered in slots 0.., and raises the thresholds. NPL * 64 >= c.cnt.
template <int NPL>
__device__ __forceinline__ void cand_reduce(Cands &c, int k, int cap, int lane) {
  wave_lds_sync();
  uint64_t v[NPL];
#pragma unroll
  for (int i = 0; i < NPL; i++) {
    const int j = lane + i * kWave;
    v[i] = j < c.cnt ? c.buf[j] : 0;
  }
  const uint64_t t = select_threshold<NPL>(v, k, cap);
  wave_lds_sync();
  c.cnt = wave_store_ge<NPL>(c.buf, v, t, lane);
  if (t > c.kmin) {
    c.kmin = t;
    c.vmin = from_order_bits((uint32_t)(t >> 32));
  }
  wave_lds_sync();
}

__device__ __forceinline__ void cand_reduce_any(Cands &c, int k, int cap, int lane) {
  if (c.cnt <= kWave) cand_reduce<1>(c, k, cap, lane);
  else if (c.cnt <= 2 * kWave) cand_reduce<2>(c, k, cap, lane);
  else cand_reduce<kCandPerLane>(c, k, cap, lane);
}

// Buffer overflow (rare once the thresholds are seeded): keep at most kKeep.
__device__ __forceinline__ void cand_compact(Cands &c, int k, int lane) {
  cand_reduce<kCandPerLane>(c, k, kKeep, lane);
}

// Initial thresholds from the first round: the k-th largest of the lanes'
// maxima (each an actual logit), so at least k of the wave's logits are at or
// above it and nothing below it can be among the wave's k best.
__device__ __forceinline__ void cand_seed(Cands &c, float lane_max, int k) {
  const uint32_t ob = order_bits(lane_max);
  const bool ok = lane_max > kNegInf;
  if (__popcll(__ballot(ok)) < k) return;
  uint32_t t = 0;
  for (int b = 31; b >= 0; b--) {
    const uint32_t cb = t | (1u << b);
    if (__popcll(__ballot(ok && ob >= cb)) >= k) t = cb;
  }
  c.kmin = (uint64_t)t << 32;
  c.vmin = from_order_bits(t);
}

// Offers up to 8 logits per lane (elements e < nvalid, ids id0 + e). Only
// logits at or above vmin are looked at, one per lane per iteration.
__device__ __forceinline__ void cand_offer(Cands &c, int k, int lane, const float (&x)[8], uint32_t id0,
                                           int nvalid) {
  uint32_t m = 0;
#pragma unroll
  for (int e = 0; e < 8; e++) m |= ((e < nvalid) & (x[e] >= c.vmin)) ? (1u << e) : 0u;
  const uint64_t below = (1ull << lane) - 1ull;
  while (__any(m != 0)) {
    const int e = m ? __builtin_ctz(m) : 0;
    float xv = x[0];
#pragma unroll
    for (int q = 1; q < 8; q++) xv = e == q ? x[q] : xv;
    const uint64_t key = m ? cand_key(xv, id0 + (uint32_t)e) : 0;
    bool take = key != 0 && key >= c.kmin;
    uint64_t b = __ballot(take);
    if (c.cnt + __popcll(b) > kCandCap) {
      cand_compact(c, k, lane);
      take = key != 0 && key >= c.kmin;
      b = __ballot(take);
    }
    if (take) c.buf[c.cnt + __popcll(b & below)] = key;
    c.cnt += __popcll(b);
    m &= m - 1u;
  }
}

// Philox4x64-10 (Salmon et al., SC 2011): first output word.
__device__ __forceinline__ uint64_t philox_w0(uint64_t c0, uint64_t c1, uint64_t k0, uint64_t k1) {
  uint64_t c2 = 0, c3 = 0;
#pragma unroll
  for (int r = 0; r < 10; r++) {
    const uint64_t m0 = 0xD2E7470EE14C6C93ull, m1 = 0xCA5A826395121157ull;
    const uint64_t lo0 = m0 * c0, hi0 = __umul64hi(m0, c0);
    const uint64_t lo1 = m1 * c2, hi1 = __umul64hi(m1, c2);
    const uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
    k0 += 0x9E3779B97F4A7C15ull;
    k1 += 0xBB67AE8584CAA73Bull;
  }
  return c0;
}

// The draw of one row by one wave from its k best candidate keys win[0 ..
// nwin) (unordered; nwin <= kTopKMax, 0 = empty): keys sorted descending by
// rank counting into `sorted`, the temperature softmax over them relative to
// the largest, the shortest prefix reaching top_p of the mass, and the
// inverse-CDF draw with u = top 24 bits of Philox4x64-10 at counter (step,
// row, 0, 0), key (seed, 0). Writes p.tokens[row].
__device__ __forceinline__ void sample_draw(const EntropyParams &p, int row, int lane, uint64_t *win,
                                            uint64_t *sorted, int nwin) {
  wave_lds_sync();
  const uint64_t key = lane < nwin ? win[lane] : 0;
  int rank = 0;
  for (int j = 0; j < nwin; j++) rank += win[j] > key;
  if (lane < nwin) sorted[rank] = key;
  wave_lds_sync();
  const uint64_t mine = lane < nwin ? sorted[lane] : 0;
  const bool live = mine != 0;  // lanes 0 .. nwin - 1
  const float xr = live ? from_order_bits((uint32_t)(mine >> 32)) : kNegInf;
  const uint32_t id = ~(uint32_t)(mine & 0xffffffffu);
  const float x0 = __shfl(xr, 0, kWave);
  const float cexp = p.inv_t * kLog2e;
  float e = live ? fast_exp2((xr - x0) * cexp) : 0.f;
  if (!(e >= 0.f)) e = 0.f;  // -inf - (-inf) and similar never reach a live lane; belt and braces
  // Inclusive prefix sum over lanes.
  float cum = e;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const float o = __shfl_up(cum, off, kWave);
    if (lane >= off) cum += o;
  }
  const uint64_t livemask = __ballot(live);
  const int nlive = __popcll(livemask);
  const float Z = __shfl(cum, nlive - 1, kWave);
  int keep = nlive;
  if (p.top_p < 1.0f) {
    const uint64_t reach = __ballot(live && cum >= p.top_p * Z);
    if (reach) keep = __ffsll((long long)reach);  // lowest lane + 1
  }
  const float mass = __shfl(cum, keep - 1, kWave);
  const uint64_t w0 = philox_w0(p.step, (uint64_t)row, p.seed, 0);
  const float u = (float)(w0 >> 40) * (1.0f / 16777216.0f);
  const float target = u * mass;
  const uint64_t over = __ballot(lane < keep && cum > target);
  const int pick = over ? __ffsll((long long)over) - 1 : keep - 1;
  const uint32_t tok = __shfl(id, pick, kWave);
  if (lane == 0) p.tokens[row] = (int32_t)tok;
}

// Bytes of LDS a sampling row wave uses: its candidate buffer and the sorted
// k best.
constexpr size_t kSampleRowLds = (size_t)(kCandCap + kTopKMax) * sizeof(uint64_t);

// One whole logit row by one wave with the sampler: the entropy and detector
// of entropy_row_wave, the row's k best logits collected into the wave's
// candidate buffer as the row streams (thresholds seeded from the lane maxima
// of the first bank), then the draw. Two banks of U vector loads, as there.
// lds: kSampleRowLds bytes of LDS owned by the wave.
template <typename T, int U>
__device__ __forceinline__ void entropy_sample_row_wave(const EntropyParams &p, int row, int lane, uint64_t *lds) {
  const T *x = static_cast<const T *>(p.logits) + (size_t)row * p.ld;
  const float c = p.inv_temp * kLog2e;
  const int nvec = p.V / 8;
  const rsrc_t rr = row_rsrc(x, (uint32_t)nvec * 8u * (uint32_t)sizeof(T));
  constexpr int BANK = U * kWave;  // vectors per bank
  Cands cs{lds, 0, 1, kNegInf};
  Tri t{kNegInf, 0.f, 0.f};
  Vec8<T> a[U], b[U];
#pragma unroll
  for (int u = 0; u < U; u++) a[u].load(rr, u * kWave + lane);
  {
    float mx = kNegInf;
#pragma unroll
    for (int u = 0; u < U; u++) {
      float y[8];
      a[u].get(y);
      if (u * kWave + lane < nvec)
#pragma unroll
        for (int e = 0; e < 8; e++) mx = vmax(mx, y[e]);
    }
    cand_seed(cs, mx, p.top_k);
  }
  // Every lane offers in lockstep (vectors past the row offer nothing).
  auto fold = [&](const Vec8<T> &w, int v) {
    float y[8];
    w.get(y);
    const bool ok = v < nvec;
    cand_offer(cs, p.top_k, lane, y, (uint32_t)v * 8u, ok ? 8 : 0);
    if (ok) tri_fold8(t, y, c);
  };
  for (int v0 = 0; v0 < nvec; v0 += 2 * BANK) {
#pragma unroll
    for (int u = 0; u < U; u++) b[u].load(rr, v0 + BANK + u * kWave + lane);
#pragma unroll
    for (int u = 0; u < U; u++) fold(a[u], v0 + u * kWave + lane);
    if (v0 + BANK >= nvec) break;
#pragma unroll
    for (int u = 0; u < U; u++) a[u].load(rr, v0 + 2 * BANK + u * kWave + lane);
#pragma unroll
    for (int u = 0; u < U; u++) fold(b[u], v0 + BANK + u * kWave + lane);
  }
  {
    // The V % 8 trailing logits, one per lane.
    const int e = nvec * 8 + lane;
    float y[8] = {kNegInf, kNegInf, kNegInf, kNegInf, kNegInf, kNegInf, kNegInf, kNegInf};
    const bool has = e < p.V;
    if (has) y[0] = load1(x + e);
    cand_offer(cs, p.top_k, lane, y, (uint32_t)e, has ? 1 : 0);
    if (has) {
      float z[1] = {y[0] * c};
      tri_add<1>(t, z);
    }
  }
#pragma unroll
  for (int msk = 32; msk >= 1; msk >>= 1) {
    Tri o{shfl_xor(t.m, msk), shfl_xor(t.z, msk), shfl_xor(t.s, msk)};
    t = tri_merge(t, o);
  }
  const float H = finish_entropy(t);
  if (lane == 0) p.H[row] = H;
  detector_push(p, row, H, lane);
  if (cs.cnt > p.top_k) cand_reduce_any(cs, p.top_k, p.top_k, lane);  // exactly the k best
  sample_draw(p, row, lane, cs.buf, lds + kCandCap, cs.cnt);
}

}  // namespace
}  // namespace kvr
