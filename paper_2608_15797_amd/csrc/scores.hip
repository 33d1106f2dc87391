// Window re-computation of the accumulated-attention importance score
// (Sec. 2.1): for the last nq tokens of every sequence, window row r attends
// causally over len - (nq-1-r) cache entries; each entry's score is the
// probability mass it receives, summed over the window rows and over the G
// query heads of its KV head. This runs when a whole step's tokens are encoded
// in one pass (a committed helper step, a one-shot prompt), not per decoded
// token.
//
// bf16 caches: the R = G * nq window rows of one (sequence, layer, KV head)
// form a dense [R x D] x [D x n] contraction, done on MFMA
// (v_mfma_f32_16x16x16bf16_1k, rows in the M dimension, keys in N). One
// workgroup of four waves per (sequence, layer, KV head); each wave takes two
// 16-row blocks at a time and makes two passes over the keys: the first builds
// every row's softmax maximum and normaliser (online, per lane, then merged
// across the 16 lanes holding the same rows), the second recomputes the
// logits, forms the probabilities and adds their column sums into an LDS
// accumulator. The head's scores are written (or added) once at the end, so
// the result does not depend on the order the waves finish in.
//
// The contraction index d is dealt to lanes so that each lane reads one
// contiguous quarter of a row: in k-step t, operand element i of lane group
// q = lane / 16 is d = q * D/4 + 4 t + i, for the q rows (A) and the keys (B)
// alike.
//
// float32 caches take a plain one-wave-per-head kernel (one key per lane).
#include <hip/hip_runtime.h>

#include "kvr_device.h"
#include "kvr_internal.h"

namespace kvr {

namespace {

template <typename T>
__device__ __forceinline__ float ld(const T *p, size_t i);
template <>
__device__ __forceinline__ float ld<float>(const float *p, size_t i) { return p[i]; }
template <>
__device__ __forceinline__ float ld<bf16_t>(const bf16_t *p, size_t i) { return bf16_to_f32(p[i]); }

template <typename T>
__global__ __launch_bounds__(64) void window_scores_kernel(ScoreParams p) {
  extern __shared__ float smem[];
  const int unit = blockIdx.x;
  const int h = unit % p.Hkv;
  const int sl = unit / p.Hkv;
  const int l = sl % p.L;
  const int s = sl / p.L;
  const int lane = threadIdx.x;
  const int D = p.D, G = p.G;
  int n = p.len[s];
  n = n < 0 ? 0 : (n > p.cap ? p.cap : n);
  const T *K = static_cast<const T *>(p.k) + (size_t)unit * p.cap * D;
  float *qs = smem;          // [D]
  float *xs = smem + D;      // [cap]
  float *acc = xs + p.cap;   // [cap]
  for (int j = lane; j < n; j += kWave) acc[j] = 0.f;
  const float sl2 = p.scale * kLog2e;
  for (int r = 0; r < p.nq; r++) {
    const int nr = n - (p.nq - 1 - r);
    if (nr <= 0) continue;
    for (int g = 0; g < G; g++) {
      const size_t qoff = ((((size_t)s * p.L + l) * p.Hq + h * G + g) * p.nq + r) * D;
      __syncthreads();
      for (int d = lane; d < D; d += kWave) qs[d] = ld<T>(static_cast<const T *>(p.q_win), qoff + d);
      __syncthreads();
      float mloc = -__builtin_huge_valf();
      for (int j = lane; j < nr; j += kWave) {
        float dot = 0.f;
        for (int d = 0; d < D; d++) dot = fmaf(qs[d], ld<T>(K, (size_t)j * D + d), dot);
        xs[j] = dot * sl2;
        mloc = fmaxf(mloc, xs[j]);
      }
      const float m = wave_max(mloc);
      float zloc = 0.f;
      for (int j = lane; j < nr; j += kWave) zloc += fast_exp2(xs[j] - m);
      const float iz = 1.0f / wave_sum(zloc);
      for (int j = lane; j < nr; j += kWave) acc[j] += fast_exp2(xs[j] - m) * iz;
    }
  }
  float *sc = p.scores + (size_t)unit * p.cap;
  for (int j = lane; j < n; j += kWave) sc[j] = p.accumulate ? sc[j] + acc[j] : acc[j];
}


typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ rsrc_t make_rsrc(const void *ptr, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(ptr), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ short4_t s4(uint32_t a, uint32_t b) {
  const uint32_t v[2] = {a, b};
  return __builtin_bit_cast(short4_t, v);
}

constexpr float kNegInf = -__builtin_huge_valf();

template <int D>
struct WGeo {
  static constexpr int QD = D / 4;   // elements per lane quarter of a row
  static constexpr int KS = D / 16;  // MFMA k-steps over D
  static constexpr int NV = QD / 8;  // 16-byte vectors per quarter
};

// Quarter q of row `row` of a [rows][D] bf16 array; zero past the resource.
template <int D>
__device__ __forceinline__ void load_quarter(rsrc_t r, int row, int q, u32x4 (&v)[WGeo<D>::NV]) {
  const uint32_t off = ((uint32_t)row * D + (uint32_t)q * WGeo<D>::QD) * 2u;
#pragma unroll
  for (int i = 0; i < WGeo<D>::NV; i++) v[i] = __builtin_amdgcn_raw_buffer_load_b128(r, off + 16u * i, 0, 0);
}

// Operand of k-step t from a loaded quarter: elements 4t .. 4t+3.
template <int D>
__device__ __forceinline__ short4_t kstep_op(const u32x4 (&v)[WGeo<D>::NV], int t) {
  const u32x4 w = v[t >> 1];
  return (t & 1) ? s4(w.z, w.w) : s4(w.x, w.y);
}

constexpr int kRB = 2;  // 16-row blocks per wave at a time

template <int D>
__device__ __forceinline__ void logits_tile(const short4_t (&qa)[kRB][WGeo<D>::KS],
                                            const u32x4 (&kv)[WGeo<D>::NV], float4_t (&c)[kRB]) {
#pragma unroll
  for (int b = 0; b < kRB; b++) c[b] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int t = 0; t < WGeo<D>::KS; t++) {
    const short4_t kb = kstep_op<D>(kv, t);
#pragma unroll
    for (int b = 0; b < kRB; b++) c[b] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(qa[b][t], kb, c[b], 0, 0, 0);
  }
}

template <int D>
__global__ __launch_bounds__(256) void window_scores_bf16(ScoreParams p) {
  extern __shared__ float acc[];  // [cap]
  const int unit = blockIdx.x;
  const int h = unit % p.Hkv;
  const int sl = unit / p.Hkv;
  const int l = sl % p.L;
  const int s = sl / p.L;
  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  const int lane = tid % kWave;
  const int gq = lane >> 4, col = lane & 15;
  int n = p.len[s];
  n = n < 0 ? 0 : (n > p.cap ? p.cap : n);
  for (int j = tid; j < n; j += blockDim.x) acc[j] = 0.f;
  __syncthreads();

  const int R = p.G * p.nq;
  const bf16_t *Q = static_cast<const bf16_t *>(p.q_win) + (((size_t)s * p.L + l) * p.Hq + (size_t)h * p.G) * p.nq * D;
  const bf16_t *K = static_cast<const bf16_t *>(p.k) + (size_t)unit * p.cap * D;
  const rsrc_t qr = make_rsrc(Q, (uint32_t)R * D * 2u);
  const rsrc_t kr = make_rsrc(K, (uint32_t)n * D * 2u);
  const float c = p.scale * kLog2e;
  const int tiles = (n + 15) / 16;
  const int blocks = (R + 15) / 16;

  for (int rb = wave * kRB; rb < blocks; rb += 4 * kRB) {
    short4_t qa[kRB][WGeo<D>::KS];
    int nr[kRB][4];
#pragma unroll
    for (int b = 0; b < kRB; b++) {
      u32x4 v[WGeo<D>::NV];
      load_quarter<D>(qr, (rb + b) * 16 + col, gq, v);
#pragma unroll
      for (int t = 0; t < WGeo<D>::KS; t++) qa[b][t] = kstep_op<D>(v, t);
#pragma unroll
      for (int i = 0; i < 4; i++) {
        const int row = (rb + b) * 16 + 4 * gq + i;  // output row of this lane
        const int r = row % p.nq;
        nr[b][i] = row < R ? n - (p.nq - 1 - r) : 0;
      }
    }
    // Pass 1: per-row maximum and normaliser over the visible keys.
    float m[kRB][4], z[kRB][4];
#pragma unroll
    for (int b = 0; b < kRB; b++)
#pragma unroll
      for (int i = 0; i < 4; i++) { m[b][i] = kNegInf; z[b][i] = 0.f; }
    u32x4 kv[WGeo<D>::NV];
    if (tiles > 0) load_quarter<D>(kr, col, gq, kv);
    for (int kt = 0; kt < tiles; kt++) {
      u32x4 cur[WGeo<D>::NV];
#pragma unroll
      for (int i = 0; i < WGeo<D>::NV; i++) cur[i] = kv[i];
      if (kt + 1 < tiles) load_quarter<D>(kr, (kt + 1) * 16 + col, gq, kv);
      float4_t cc[kRB];
      logits_tile<D>(qa, cur, cc);
      const int j = kt * 16 + col;
#pragma unroll
      for (int b = 0; b < kRB; b++)
#pragma unroll
        for (int i = 0; i < 4; i++) {
          if (j < nr[b][i]) {
            const float x = cc[b][i] * c;
            if (x > m[b][i]) {
              z[b][i] = z[b][i] * fast_exp2(m[b][i] - x) + 1.f;
              m[b][i] = x;
            } else {
              z[b][i] += fast_exp2(x - m[b][i]);
            }
          }
        }
    }
    // Merge the 16 lanes that hold the same rows (lane bits 0..3).
#pragma unroll
    for (int msk = 1; msk <= 8; msk <<= 1)
#pragma unroll
      for (int b = 0; b < kRB; b++)
#pragma unroll
        for (int i = 0; i < 4; i++) {
          const float om = shfl_xor(m[b][i], msk);
          const float oz = shfl_xor(z[b][i], msk);
          const float M = fmaxf(m[b][i], om);
          float zz = 0.f;
          if (z[b][i] > 0.f) zz += z[b][i] * fast_exp2(m[b][i] - M);
          if (oz > 0.f) zz += oz * fast_exp2(om - M);
          m[b][i] = M;
          z[b][i] = zz;
        }
    float iz[kRB][4];
#pragma unroll
    for (int b = 0; b < kRB; b++)
#pragma unroll
      for (int i = 0; i < 4; i++) iz[b][i] = z[b][i] > 0.f ? 1.0f / z[b][i] : 0.f;
    // Pass 2: probabilities, column sums into the LDS accumulator.
    if (tiles > 0) load_quarter<D>(kr, col, gq, kv);
    for (int kt = 0; kt < tiles; kt++) {
      u32x4 cur[WGeo<D>::NV];
#pragma unroll
      for (int i = 0; i < WGeo<D>::NV; i++) cur[i] = kv[i];
      if (kt + 1 < tiles) load_quarter<D>(kr, (kt + 1) * 16 + col, gq, kv);
      float4_t cc[kRB];
      logits_tile<D>(qa, cur, cc);
      const int j = kt * 16 + col;
      float cs = 0.f;
#pragma unroll
      for (int b = 0; b < kRB; b++)
#pragma unroll
        for (int i = 0; i < 4; i++)
          if (j < nr[b][i] && iz[b][i] > 0.f) cs += fast_exp2(cc[b][i] * c - m[b][i]) * iz[b][i];
      cs += shfl_xor(cs, 16);
      cs += shfl_xor(cs, 32);
      if (gq == 0 && j < n) atomicAdd(&acc[j], cs);
    }
  }
  __syncthreads();
  float *sc = p.scores + (size_t)unit * p.cap;
  for (int j = tid; j < n; j += blockDim.x) sc[j] = p.accumulate ? sc[j] + acc[j] : acc[j];
}

}  // namespace

hipError_t launch_accumulate_scores(const ScoreParams &p, hipStream_t stream) {
  const dim3 grid(p.S * p.L * p.Hkv);
  if (p.dtype == 0) {
    const size_t lds = ((size_t)p.D + 2 * (size_t)p.cap) * sizeof(float);
    hipLaunchKernelGGL(window_scores_kernel<float>, grid, dim3(64), lds, stream, p);
  } else {
    const size_t lds = (size_t)p.cap * sizeof(float);
    if (p.D == 128) hipLaunchKernelGGL(window_scores_bf16<128>, grid, dim3(256), lds, stream, p);
    else hipLaunchKernelGGL(window_scores_bf16<64>, grid, dim3(256), lds, stream, p);
  }
  return hipGetLastError();
}

}  // namespace kvr
