// Redundancy-aware eviction score (App. C, KV eviction: query-attention
// importance mixed with key redundancy by cosine similarity, weight lambda,
// with pooling; App. D.3). Per (sequence, layer, KV head) of a sequence that
// evicts this step, over its candidates c < m = n - W:
//   P_c  = max of the importance over candidates within pool/2 slots of c;
//   R_c  = mean cosine similarity of key c to the other candidates;
//   out_c = lam * P_c / sum P - (1 - lam) * softmax(R)_c.
//
// The mean cosine needs no m x m Gram matrix: with u_c = k_c / |k_c| and
// s = sum_c u_c, sum_{c' != c} cos(k_c, k_c') = u_c . s - 1 (0 - 0 for a zero
// key), so two streaming passes over the candidate keys suffice: one for the
// norms and s, one for u_c . s. One 256-thread workgroup per head; each row is
// read by D/8 lanes of 8 elements (bf16, D = 128: 16 lanes x 16 bytes, four rows
// per wave instruction), and the head's importance, norms and R stay in LDS. Everything a head needs is
// read before its output is written, so `out` may be the importance array.
#include <hip/hip_runtime.h>

#include "kvr_device.h"
#include "kvr_internal.h"

namespace kvr {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;

template <typename T>
struct Row8;  // 8 elements of a row as floats
template <>
struct Row8<bf16_t> {
  static __device__ __forceinline__ void load(const bf16_t *p, float (&x)[8]) {
    const u32x4 w = *reinterpret_cast<const u32x4 *>(p);
    x[0] = bf16_lo(w.x); x[1] = bf16_hi(w.x); x[2] = bf16_lo(w.y); x[3] = bf16_hi(w.y);
    x[4] = bf16_lo(w.z); x[5] = bf16_hi(w.z); x[6] = bf16_lo(w.w); x[7] = bf16_hi(w.w);
  }
};
template <>
struct Row8<float> {
  static __device__ __forceinline__ void load(const float *p, float (&x)[8]) {
    const u32x4 a = reinterpret_cast<const u32x4 *>(p)[0];
    const u32x4 b = reinterpret_cast<const u32x4 *>(p)[1];
    x[0] = __uint_as_float(a.x); x[1] = __uint_as_float(a.y); x[2] = __uint_as_float(a.z); x[3] = __uint_as_float(a.w);
    x[4] = __uint_as_float(b.x); x[5] = __uint_as_float(b.y); x[6] = __uint_as_float(b.z); x[7] = __uint_as_float(b.w);
  }
};

__device__ __forceinline__ float block_reduce(float v, float *red, bool is_max) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const float o = shfl_xor(v, m);
    v = is_max ? fmaxf(v, o) : v + o;
  }
  const int wave = threadIdx.x / kWave;
  __syncthreads();
  if ((threadIdx.x & (kWave - 1)) == 0) red[wave] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int w = 1; w < kWaves; w++) r = is_max ? fmaxf(r, red[w]) : r + red[w];
  return r;
}

// D = 64 or 128 elements per row, read as D/8 lanes x 8 elements; a wave
// covers 64 / (D/8) rows per instruction.
template <typename T, int D>
__global__ __launch_bounds__(kThreads) void redundancy_kernel(RedundancyParams p) {
  extern __shared__ float lds[];
  constexpr int LPR = D / 8;            // lanes per row
  constexpr int RPW = kWave / LPR;      // rows per wave instruction
  const int unit = blockIdx.x;          // ((s * L) + l) * Hkv + h
  const int s = unit / (p.L * p.Hkv);
  int n = p.len[s];
  if (n <= p.B + p.buffer) return;
  if (n > p.cap) n = p.cap;
  const int m = n - p.W;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int sub = lane / LPR;           // row within the wave instruction
  const int part = lane % LPR;          // 8-element slice of the row

  float *imp = lds;                     // [cap] importance, then pooled
  float *nrm = imp + p.cap;             // [cap] 1 / |k_c| (0 for a zero key)
  float *red_s = nrm + p.cap;           // [kWaves][D] partial sums of u
  float *svec = red_s + kWaves * D;     // [D] s = sum u_c
  float *red = svec + D;                // [kWaves] reduction scratch
  float *R = red + kWaves;              // [cap]

  const T *K = static_cast<const T *>(p.k) + (size_t)unit * p.cap * D;
  const float *I = p.importance + (size_t)unit * p.cap;
  float *out = p.out + (size_t)unit * p.cap;
  for (int c = tid; c < m; c += kThreads) imp[c] = I[c];

  // Pass 1: norms and the partial sums of the unit keys.
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int c0 = wave * RPW; c0 < m; c0 += kWaves * RPW) {
    const int c = c0 + sub;
    float x[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (c < m) Row8<T>::load(K + (size_t)c * D + part * 8, x);
    float sq = 0.f;
#pragma unroll
    for (int e = 0; e < 8; e++) sq = fmaf(x[e], x[e], sq);
    // Row norm: reduce over the LPR lanes of this row.
#pragma unroll
    for (int mk = 1; mk < LPR; mk <<= 1) sq += shfl_xor(sq, mk);
    const float inv = sq > 0.f ? 1.0f / sqrtf(sq) : 0.f;
    if (c < m && part == 0) nrm[c] = inv;
#pragma unroll
    for (int e = 0; e < 8; e++) acc[e] = fmaf(x[e], inv, acc[e]);
  }
  // Sum the slices of the wave's row groups, then the waves.
#pragma unroll
  for (int e = 0; e < 8; e++)
#pragma unroll
    for (int mk = LPR; mk < kWave; mk <<= 1) acc[e] += shfl_xor(acc[e], mk);
  if (sub == 0)
#pragma unroll
    for (int e = 0; e < 8; e++) red_s[wave * D + part * 8 + e] = acc[e];
  __syncthreads();
  for (int d = tid; d < D; d += kThreads) {
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; w++) v += red_s[w * D + d];
    svec[d] = v;
  }
  __syncthreads();

  // Pass 2: R_c = (u_c . s - [k_c != 0]) / (m - 1).
  float sv[8];
#pragma unroll
  for (int e = 0; e < 8; e++) sv[e] = svec[part * 8 + e];
  const float inv_m1 = m > 1 ? 1.0f / (float)(m - 1) : 0.f;
  for (int c0 = wave * RPW; c0 < m; c0 += kWaves * RPW) {
    const int c = c0 + sub;
    float x[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (c < m) Row8<T>::load(K + (size_t)c * D + part * 8, x);
    float dot = 0.f;
#pragma unroll
    for (int e = 0; e < 8; e++) dot = fmaf(x[e], sv[e], dot);
#pragma unroll
    for (int mk = 1; mk < LPR; mk <<= 1) dot += shfl_xor(dot, mk);
    if (c < m && part == 0) {
      const float iv = nrm[c];
      R[c] = iv > 0.f ? (dot * iv - 1.0f) * inv_m1 : 0.f;
    }
  }
  __syncthreads();

  // Pooled importance, staged in `out` (this head's importance is in LDS and
  // its keys are read, so the output may overwrite the importance array).
  const int r = p.pool / 2;
  float psum = 0.f, rmax = -__builtin_huge_valf();
  for (int c = tid; c < m; c += kThreads) {
    float v = imp[c];
    const int lo = c - r < 0 ? 0 : c - r, hi = c + r >= m ? m - 1 : c + r;
    for (int j = lo; j <= hi; j++) v = fmaxf(v, imp[j]);
    psum += v;
    rmax = fmaxf(rmax, R[c]);
    out[c] = v;
  }
  const float Psum = block_reduce(psum, red, false);
  const float Rmax = block_reduce(rmax, red, true);
  float esum = 0.f;
  for (int c = tid; c < m; c += kThreads) esum += fast_exp2((R[c] - Rmax) * kLog2e);
  const float Esum = block_reduce(esum, red, false);
  const float lam = p.lam;
  const float ip = Psum > 0.f ? 1.0f / Psum : 0.f;
  const float ie = 1.0f / Esum;
  for (int c = tid; c < m; c += kThreads) {
    const float ih = Psum > 0.f ? out[c] * ip : 1.0f / (float)m;
    const float rh = fast_exp2((R[c] - Rmax) * kLog2e) * ie;
    out[c] = lam * ih - (1.0f - lam) * rh;
  }
}

}  // namespace

size_t redundancy_lds_bytes(int cap, int D) {
  return ((size_t)3 * cap + (size_t)(kWaves + 1) * D + kWaves) * sizeof(float);
}

hipError_t launch_redundancy(const RedundancyParams &p, hipStream_t stream) {
  const dim3 grid(p.S * p.L * p.Hkv);
  const size_t lds = redundancy_lds_bytes(p.cap, p.D);
  if (p.dtype == 0) {
    if (p.D == 128) hipLaunchKernelGGL((redundancy_kernel<float, 128>), grid, dim3(kThreads), lds, stream, p);
    else hipLaunchKernelGGL((redundancy_kernel<float, 64>), grid, dim3(kThreads), lds, stream, p);
  } else {
    if (p.D == 128) hipLaunchKernelGGL((redundancy_kernel<bf16_t, 128>), grid, dim3(kThreads), lds, stream, p);
    else hipLaunchKernelGGL((redundancy_kernel<bf16_t, 64>), grid, dim3(kThreads), lds, stream, p);
  }
  return hipGetLastError();
}

}  // namespace kvr
