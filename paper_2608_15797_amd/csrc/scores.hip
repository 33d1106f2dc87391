// Window re-computation of the accumulated-attention importance score
// (Sec. 2.1): for the last nq tokens of every sequence, window row r attends
// causally over len - (nq-1-r) cache entries; each entry's score is the
// probability mass it receives, summed over the window rows and over the G
// query heads of its KV head. One 64-lane wave per (sequence, layer, KV head):
// lanes own keys, q rows are staged in LDS, scores accumulate in LDS and are
// written (or added) once at the end. This runs when a whole step's tokens are
// encoded in one pass, not per decoded token, so it favours simplicity.
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

}  // namespace

hipError_t launch_accumulate_scores(const ScoreParams &p, hipStream_t stream) {
  const size_t lds = ((size_t)p.D + 2 * (size_t)p.cap) * sizeof(float);
  if (p.dtype == 0)
    hipLaunchKernelGGL(window_scores_kernel<float>, dim3(p.S * p.L * p.Hkv), dim3(64), lds, stream, p);
  else
    hipLaunchKernelGGL(window_scores_kernel<bf16_t>, dim3(p.S * p.L * p.Hkv), dim3(64), lds, stream, p);
  return hipGetLastError();
}

}  // namespace kvr
