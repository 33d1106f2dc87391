// Device-side pieces of the full-vocabulary entropy (Eq. (4)) and its
// moving-average detector (Sec. 3.2) shared by the entropy kernels and the
// base-attention launch that computes the step's entropies alongside.
//
// Each lane keeps an online triple in the log2 domain: m = reference maximum
// of y = inv_temp * x * log2(e), Z = sum 2^(y - m) and S = sum (y - m) 2^(y - m),
// rescaled when the reference moves. Since the natural-log entropy is
// H = ln Z - (sum (x' - m') e^(x' - m')) / Z with x' the scaled logits, in log2
// units H = ln2 * (log2 Z - S / Z). Triples merge associatively.
#pragma once

#include <hip/hip_runtime.h>

#include "kvr_device.h"
#include "kvr_internal.h"

namespace kvr {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();

struct Tri {
  float m, z, s;
};

__device__ __forceinline__ Tri tri_merge(Tri a, Tri b) {
  const float M = fmaxf(a.m, b.m);
  if (M == kNegInf) return Tri{kNegInf, 0.f, 0.f};
  Tri r{M, 0.f, 0.f};
  if (a.z > 0.f) {
    const float f = fast_exp2(a.m - M);
    r.z += a.z * f;
    r.s += (a.s + (a.m - M) * a.z) * f;
  }
  if (b.z > 0.f) {
    const float f = fast_exp2(b.m - M);
    r.z += b.z * f;
    r.s += (b.s + (b.m - M) * b.z) * f;
  }
  return r;
}

// Fold a group of already scaled values (log2 domain) into the triple.
template <int N>
__device__ __forceinline__ void tri_add(Tri &t, const float (&y)[N]) {
  float lm = y[0];
#pragma unroll
  for (int e = 1; e < N; e++) lm = fmaxf(lm, y[e]);
  if (lm > t.m) {
    if (t.z > 0.f) {
      const float f = fast_exp2(t.m - lm);
      t.s = (t.s + (t.m - lm) * t.z) * f;
      t.z *= f;
    }
    t.m = lm;
  }
#pragma unroll
  for (int e = 0; e < N; e++) {
    // Clamp keeps (-inf) - m and (-inf) - (-inf) finite so 0 * d stays 0.
    const float d = fmaxf(y[e] - t.m, -256.0f);
    const float w = fast_exp2(d);
    t.z += w;
    t.s = fmaf(d, w, t.s);
  }
}

typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ rsrc_t row_rsrc(const void *p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes, 0x00020000);
}

// Eight logits of a row, held as the raw loaded words until they are used, so
// that a round's loads cost 4 (bf16) or 8 (fp32) registers per vector.
template <typename T>
struct Vec8;
template <>
struct Vec8<bf16_t> {
  u32x4 w;
  __device__ __forceinline__ void load(rsrc_t r, int v) {
    w = __builtin_amdgcn_raw_buffer_load_b128(r, (uint32_t)v * 16u, 0, kStreamLoad);
  }
  __device__ __forceinline__ void get(float (&y)[8]) const {
    y[0] = bf16_lo(w.x); y[1] = bf16_hi(w.x); y[2] = bf16_lo(w.y); y[3] = bf16_hi(w.y);
    y[4] = bf16_lo(w.z); y[5] = bf16_hi(w.z); y[6] = bf16_lo(w.w); y[7] = bf16_hi(w.w);
  }
};
template <>
struct Vec8<float> {
  u32x4 a, b;
  __device__ __forceinline__ void load(rsrc_t r, int v) {
    a = __builtin_amdgcn_raw_buffer_load_b128(r, (uint32_t)v * 32u, 0, kStreamLoad);
    b = __builtin_amdgcn_raw_buffer_load_b128(r, (uint32_t)v * 32u + 16u, 0, kStreamLoad);
  }
  __device__ __forceinline__ void get(float (&y)[8]) const {
    y[0] = __uint_as_float(a.x); y[1] = __uint_as_float(a.y); y[2] = __uint_as_float(a.z); y[3] = __uint_as_float(a.w);
    y[4] = __uint_as_float(b.x); y[5] = __uint_as_float(b.y); y[6] = __uint_as_float(b.z); y[7] = __uint_as_float(b.w);
  }
};

// The triple's reference m may trail the running maximum by up to this much
// (log2 units, a factor of 256): every term 2^(y - m) stays finite and exact
// to fp32 rounding, and the rescale is skipped for almost every vector once
// the first few have been seen. The entropy does not depend on m.
constexpr float kSlack = 8.0f;

__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

// Fold eight raw logits x into the triple, y = c * x with c > 0.
__device__ __forceinline__ void tri_fold8(Tri &t, const float (&x)[8], float c) {
  // NaN-propagating maximum: no operand canonicalisation, three-input
  // instructions (NaN logits are unsupported anyway).
  const float lm = vmax(vmax(vmax(x[0], x[1]), vmax(x[2], x[3])), vmax(vmax(x[4], x[5]), vmax(x[6], x[7]))) * c;
  if (lm > t.m + kSlack) {
    if (t.z > 0.f) {
      const float f = fast_exp2(t.m - lm);
      t.s = (t.s + (t.m - lm) * t.z) * f;
      t.z *= f;
    }
    t.m = lm;
  }
  const float nm = -t.m;
#pragma unroll
  for (int e = 0; e < 8; e++) {
    // Clamp keeps -inf logits (and -inf - (-inf)) finite so 0 * d stays 0.
    const float d = fmaxf(fmaf(x[e], c, nm), -256.0f);
    const float w = fast_exp2(d);
    t.z += w;
    t.s = fmaf(d, w, t.s);
  }
}

__device__ __forceinline__ float load1(const bf16_t *ptr) { return bf16_to_f32(*ptr); }
__device__ __forceinline__ float load1(const float *ptr) { return *ptr; }

__device__ __forceinline__ float finish_entropy(Tri t) {
  return kLn2 * (log2f(t.z) - t.s / t.z);
}

// Detector update of one row by one whole wave (every lane passes the same
// H): the history entries are read by the lanes in parallel, the new entry
// taking its slot in registers, and summed with a wave reduction.
__device__ void detector_push(const EntropyParams &p, int row, float H, int lane) {
  if (!p.hist) return;
  float *h = p.hist + (size_t)row * p.window;
  const int c = p.cnt[row];
  const int slot = c % p.window;
  const int c1 = c + 1;
  const int k = c1 < p.window ? c1 : p.window;
  const bool judge = c1 >= p.guard;
  float sum = 0.f;
  if (judge) {
    for (int i = lane; i < k; i += kWave) sum += i == slot ? H : h[i];
    sum = wave_sum(sum);
  }
  if (lane == 0) {
    h[slot] = H;
    p.cnt[row] = c1;
    if (judge && sum / (float)k > p.tau) p.flag[row] = 1;
  }
}

// The set of a batch that holds global row g (uniform per workgroup).
__device__ __forceinline__ int batch_set(const EntropyBatch &b, int g) {
  int k = 0;
#pragma unroll
  for (int i = 1; i < kEntropyMaxSets; i++)
    if (i < b.nsets && g >= b.row0[i]) k = i;
  return k;
}

// Entropy (and detector update) of one whole logit row by one 64-lane wave:
// the row streams through two banks of U 16-byte vector loads per lane (the
// next bank's loads are in flight while the current one is folded), lanes
// take consecutive vectors so every load instruction reads 1 KiB, and the
// row's triple is reduced across the wave with shuffles. No partials leave
// the wave. The row must start 16-byte aligned.
template <typename T, int U>
__device__ __forceinline__ void entropy_row_wave(const EntropyParams &p, int row, int lane) {
  const T *x = static_cast<const T *>(p.logits) + (size_t)row * p.ld;
  const float c = p.inv_temp * kLog2e;
  const int nvec = p.V / 8;
  const rsrc_t rr = row_rsrc(x, (uint32_t)nvec * 8u * (uint32_t)sizeof(T));
  constexpr int BANK = U * kWave;  // vectors per bank
  Tri t{kNegInf, 0.f, 0.f};
  Vec8<T> a[U], b[U];
#pragma unroll
  for (int u = 0; u < U; u++) a[u].load(rr, u * kWave + lane);
  for (int v0 = 0; v0 < nvec; v0 += 2 * BANK) {
#pragma unroll
    for (int u = 0; u < U; u++) b[u].load(rr, v0 + BANK + u * kWave + lane);
#pragma unroll
    for (int u = 0; u < U; u++) {
      float y[8];
      a[u].get(y);
      if (v0 + u * kWave + lane < nvec) tri_fold8(t, y, c);
    }
    if (v0 + BANK >= nvec) break;
#pragma unroll
    for (int u = 0; u < U; u++) a[u].load(rr, v0 + 2 * BANK + u * kWave + lane);
#pragma unroll
    for (int u = 0; u < U; u++) {
      float y[8];
      b[u].get(y);
      if (v0 + BANK + u * kWave + lane < nvec) tri_fold8(t, y, c);
    }
  }
  // The V % 8 trailing logits, one per lane.
  const int e = nvec * 8 + lane;
  if (e < p.V) {
    float y[1] = {load1(x + e) * c};
    tri_add<1>(t, y);
  }
#pragma unroll
  for (int msk = 32; msk >= 1; msk >>= 1) {
    Tri o{shfl_xor(t.m, msk), shfl_xor(t.z, msk), shfl_xor(t.s, msk)};
    t = tri_merge(t, o);
  }
  const float H = finish_entropy(t);
  if (lane == 0) p.H[row] = H;
  detector_push(p, row, H, lane);
}

}  // namespace
}  // namespace kvr
