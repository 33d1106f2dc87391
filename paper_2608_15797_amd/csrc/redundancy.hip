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
// norms and s, one for u_c . s. The second pass takes the keys from the
// registers that the first loaded them into, up to a fixed number of rows per
// lane; only a longer head reads its remaining keys twice. One 512-thread
// workgroup per head; each row is read by D/8 lanes of 8 elements (bf16,
// D = 128: 16 lanes x 16 bytes, four rows per wave instruction), and the head's
// importance, norms and R stay in LDS. Everything a head needs is read before
// its output is written, so `out` may be the importance array.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "kvr_device.h"
#include "kvr_internal.h"

namespace kvr {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

typedef __amdgpu_buffer_rsrc_t rsrc_t;

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / kWave;
// 32-bit words of key data a lane keeps in registers from pass 1 to pass 2:
// its first kCacheWords / (words per slice) row slices are read from HBM once.
// 64 words keep the kernel within 128 registers (four waves per SIMD, two
// heads per CU) and hold 512 candidates of a bf16 D = 128 head.
constexpr int kCacheWords = 64;

// Range-checked loads: the resource covers the m candidate rows of the head,
// and a load past them returns zeros without touching memory.
__device__ __forceinline__ rsrc_t make_rsrc(const void *ptr, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(ptr), (short)0, (int)bytes, 0x00020000);
}

// 8 elements of a row (one lane's slice) as raw 32-bit words, and as floats.
template <typename T>
struct Slice {
  static constexpr int W = (int)sizeof(T) * 2;
  static __device__ __forceinline__ void load(rsrc_t r, uint32_t off, uint32_t (&w)[W]) {
#pragma unroll
    for (int i = 0; i < W / 4; i++) {
      const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, off + 16 * i, 0, 0);
      w[4 * i] = v.x; w[4 * i + 1] = v.y; w[4 * i + 2] = v.z; w[4 * i + 3] = v.w;
    }
  }
  static __device__ __forceinline__ void unpack(const uint32_t (&w)[W], float (&x)[8]) {
#pragma unroll
    for (int e = 0; e < 8; e++) {
      if constexpr (sizeof(T) == 2)
        x[e] = (e & 1) ? bf16_hi(w[e / 2]) : bf16_lo(w[e / 2]);
      else
        x[e] = __uint_as_float(w[e]);
    }
  }
};

// Sum over aligned groups of N = 8 or 16 lanes, every lane of a group getting
// the group's sum, by DPP moves within the VALU (swap neighbours, swap pairs,
// mirror the 8-lane halves, mirror the 16-lane row) instead of LDS permutes.
// Reduction (sum, or max if MAX) over aligned groups of N = 8 or 16 lanes,
// every lane of a group getting the result, by DPP moves within the VALU
// (swap neighbours, swap pairs, mirror the 8-lane halves, mirror the 16-lane
// row) instead of LDS permutes.
template <int N, bool MAX = false>
__device__ __forceinline__ float group_reduce(float v) {
  static_assert(N == 8 || N == 16, "DPP row groups");
  auto step = [](float x, auto ctrl) {
    const float o = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), decltype(ctrl)::value, 0xF, 0xF, true));
    return MAX ? fmaxf(x, o) : x + o;
  };
  v = step(v, std::integral_constant<int, 0xB1>{});   // quad_perm [1,0,3,2]
  v = step(v, std::integral_constant<int, 0x4E>{});   // quad_perm [2,3,0,1]
  v = step(v, std::integral_constant<int, 0x141>{});  // row_half_mirror
  if constexpr (N == 16) v = step(v, std::integral_constant<int, 0x140>{});  // row_mirror
  return v;
}

// Workgroup-wide sum or max: 16-lane rows by DPP, the wave's four rows by
// lane reads, then the waves through LDS.
template <bool MAX>
__device__ __forceinline__ float block_reduce(float v, float *red) {
  v = group_reduce<16, MAX>(v);
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  v = MAX ? fmaxf(fmaxf(r0, r1), fmaxf(r2, r3)) : (r0 + r1) + (r2 + r3);
  const int wave = threadIdx.x / kWave;
  __syncthreads();
  if ((threadIdx.x & (kWave - 1)) == 0) red[wave] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int w = 1; w < kWaves; w++) r = MAX ? fmaxf(r, red[w]) : r + red[w];
  return r;
}

// D = 64 or 128 elements per row, read as D/8 lanes x 8 elements; a wave
// covers 64 / (D/8) rows per instruction.
template <typename T, int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void redundancy_kernel(RedundancyParams p) {
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

  // Each wave reads row groups c_lo + i * kStep (RPW rows per group); the
  // first RC groups of a lane stay in registers for pass 2, later ones (a
  // head longer than the cache) are read again.
  using S8 = Slice<T>;
  constexpr int RC = kCacheWords / S8::W;
  constexpr int kStep = kWaves * RPW;
  const int c_lo = wave * RPW;
  const rsrc_t Kr = make_rsrc(K, (uint32_t)m * D * (uint32_t)sizeof(T));
  auto offset = [&](int c0) { return ((uint32_t)(c0 + sub) * D + part * 8) * (uint32_t)sizeof(T); };
  uint32_t kc[RC][S8::W];
#pragma unroll
  for (int i = 0; i < RC; i++) S8::load(Kr, offset(c_lo + i * kStep), kc[i]);

  // Pass 1: norms and the partial sums of the unit keys.
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  auto pass1 = [&](const float (&x)[8], int c) {
    float sq = 0.f;
#pragma unroll
    for (int e = 0; e < 8; e++) sq = fmaf(x[e], x[e], sq);
    // Row norm: reduce over the LPR lanes of this row.
    sq = group_reduce<LPR>(sq);
    const float inv = sq > 0.f ? 1.0f / sqrtf(sq) : 0.f;
    if (c < m && part == 0) nrm[c] = inv;
#pragma unroll
    for (int e = 0; e < 8; e++) acc[e] = fmaf(x[e], inv, acc[e]);
  };
#pragma unroll
  for (int i = 0; i < RC; i++) {
    // The empty asm keeps each slice's unpacking next to its use (hoisted
    // together, the unpacked floats of every slice would exceed the
    // registers).
#pragma unroll
    for (int j = 0; j < S8::W; j++) asm volatile("" : "+v"(kc[i][j])::"memory");
    float x[8];
    S8::unpack(kc[i], x);
    pass1(x, c_lo + i * kStep + sub);
  }
  for (int c0 = c_lo + RC * kStep; c0 < m; c0 += kStep) {
    uint32_t w[S8::W];
    float x[8];
    S8::load(Kr, offset(c0), w);
    S8::unpack(w, x);
    pass1(x, c0 + sub);
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
  auto pass2 = [&](const float (&x)[8], int c) {
    float dot = 0.f;
#pragma unroll
    for (int e = 0; e < 8; e++) dot = fmaf(x[e], sv[e], dot);
    dot = group_reduce<LPR>(dot);
    if (c < m && part == 0) {
      const float iv = nrm[c];
      R[c] = iv > 0.f ? (dot * iv - 1.0f) * inv_m1 : 0.f;
    }
  };
  // Groups past the cache are read again in the reverse of pass 1's order,
  // so the first reads hit the rows pass 1 read last.
  const int c_end = c_lo + RC * kStep;
  if (c_end < m)
    for (int c0 = c_end + (m - 1 - c_end) / kStep * kStep; c0 >= c_end; c0 -= kStep) {
      uint32_t w[S8::W];
      float x[8];
      S8::load(Kr, offset(c0), w);
      S8::unpack(w, x);
      pass2(x, c0 + sub);
    }
#pragma unroll
  for (int i = 0; i < RC; i++) {
    // The empty asm hides that the words are unchanged, so the compiler
    // unpacks them again here rather than keeping pass 1's floats (twice the
    // registers for bf16) alive across the passes.
#pragma unroll
    for (int j = 0; j < S8::W; j++) asm volatile("" : "+v"(kc[i][j])::"memory");
    float x[8];
    S8::unpack(kc[i], x);
    pass2(x, c_lo + i * kStep + sub);
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
  const float Psum = block_reduce<false>(psum, red);
  const float Rmax = block_reduce<true>(rmax, red);
  float esum = 0.f;
  for (int c = tid; c < m; c += kThreads) esum += fast_exp2((R[c] - Rmax) * kLog2e);
  const float Esum = block_reduce<false>(esum, red);
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
