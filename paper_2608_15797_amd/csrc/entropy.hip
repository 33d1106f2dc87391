// Full-vocabulary token entropy (Eq. (4)) with the moving-average
// degeneration detector (Sec. 3.2, implementation details), gfx950.
//
// One pass over the logits. Each thread keeps an online triple in the log2
// domain: m = running max of y = inv_temp * x * log2(e), Z = sum 2^(y - m) and
// S = sum (y - m) 2^(y - m), rescaled when m grows. Since the natural-log
// entropy is H = ln Z - (sum (x' - m') e^(x' - m')) / Z with x' the scaled
// logits, in log2 units H = ln2 * (log2 Z - S / Z). Triples merge
// associatively, first across a wave with shuffles, then across the
// workgroup's waves, then across the workgroups that split a long row: every
// split writes its triple to the workspace and the last one to finish (per-row
// atomic counter, which it resets to zero) merges them and runs the detector.
#include <hip/hip_runtime.h>

#include "kvr_device.h"
#include "kvr_internal.h"

namespace kvr {

namespace {

constexpr int kThreads = 256;
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

__device__ __forceinline__ void load8(const bf16_t *ptr, float c, float (&y)[8]) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 w = *reinterpret_cast<const u32x4 *>(ptr);
  y[0] = bf16_lo(w.x) * c; y[1] = bf16_hi(w.x) * c;
  y[2] = bf16_lo(w.y) * c; y[3] = bf16_hi(w.y) * c;
  y[4] = bf16_lo(w.z) * c; y[5] = bf16_hi(w.z) * c;
  y[6] = bf16_lo(w.w) * c; y[7] = bf16_hi(w.w) * c;
}

__device__ __forceinline__ void load8(const float *ptr, float c, float (&y)[8]) {
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  const f32x4 a = reinterpret_cast<const f32x4 *>(ptr)[0];
  const f32x4 b = reinterpret_cast<const f32x4 *>(ptr)[1];
  y[0] = a.x * c; y[1] = a.y * c; y[2] = a.z * c; y[3] = a.w * c;
  y[4] = b.x * c; y[5] = b.y * c; y[6] = b.z * c; y[7] = b.w * c;
}

__device__ __forceinline__ float load1(const bf16_t *ptr) { return bf16_to_f32(*ptr); }
__device__ __forceinline__ float load1(const float *ptr) { return *ptr; }

__device__ __forceinline__ float finish_entropy(Tri t) {
  return kLn2 * (log2f(t.z) - t.s / t.z);
}

__device__ void detector_push(const EntropyParams &p, int row, float H) {
  if (!p.hist) return;
  const int c = p.cnt[row];
  p.hist[(size_t)row * p.window + (c % p.window)] = H;
  const int c1 = c + 1;
  p.cnt[row] = c1;
  if (c1 >= p.guard) {
    const int k = c1 < p.window ? c1 : p.window;
    float sum = 0.f;
    for (int i = 0; i < k; i++) sum += p.hist[(size_t)row * p.window + i];
    if (sum / (float)k > p.tau) p.flag[row] = 1;
  }
}

// VEC = true: 16-byte loads of 8 elements (row starts 16-byte aligned).
template <typename T, bool VEC>
__global__ __launch_bounds__(kThreads) void entropy_kernel(EntropyParams p) {
  __shared__ Tri part[kThreads / kWave];
  const int row = blockIdx.y;
  const int split = blockIdx.x;
  const int splits = gridDim.x;
  const int tid = threadIdx.x;
  const T *x = static_cast<const T *>(p.logits) + (size_t)row * p.ld;
  const float c = p.inv_temp * kLog2e;

  Tri t{kNegInf, 0.f, 0.f};
  if constexpr (VEC) {
    const int nvec = p.V / 8;
    const int per = (nvec + splits - 1) / splits;
    const int v0 = split * per;
    const int v1 = min(v0 + per, nvec);
    int v = v0 + tid;
    for (; v + kThreads < v1; v += 2 * kThreads) {
      float a[8], b[8];
      load8(x + (size_t)v * 8, c, a);
      load8(x + (size_t)(v + kThreads) * 8, c, b);
      tri_add<8>(t, a);
      tri_add<8>(t, b);
    }
    if (v < v1) {
      float a[8];
      load8(x + (size_t)v * 8, c, a);
      tri_add<8>(t, a);
    }
    if (split == splits - 1) {
      const int e = nvec * 8 + tid;
      if (e < p.V) {
        float a[1] = {load1(x + e) * c};
        tri_add<1>(t, a);
      }
    }
  } else {
    const int per = (p.V + splits - 1) / splits;
    const int e0 = split * per;
    const int e1 = min(e0 + per, p.V);
    for (int e = e0 + tid; e < e1; e += kThreads) {
      float a[1] = {load1(x + e) * c};
      tri_add<1>(t, a);
    }
  }

#pragma unroll
  for (int msk = 32; msk >= 1; msk >>= 1) {
    Tri o{shfl_xor(t.m, msk), shfl_xor(t.z, msk), shfl_xor(t.s, msk)};
    t = tri_merge(t, o);
  }
  if ((tid & (kWave - 1)) == 0) part[tid / kWave] = t;
  __syncthreads();
  if (tid != 0) return;
  Tri r = part[0];
#pragma unroll
  for (int w = 1; w < kThreads / kWave; w++) r = tri_merge(r, part[w]);

  if (splits == 1) {
    const float H = finish_entropy(r);
    p.H[row] = H;
    detector_push(p, row, H);
    return;
  }
  // Cross-workgroup merge: counters [R] (padded to 16 bytes), then partials
  // [R][splits][4] floats.
  int *cnt = static_cast<int *>(p.ws);
  float *parts = reinterpret_cast<float *>(static_cast<char *>(p.ws) + (((size_t)p.R * 4 + 15) & ~(size_t)15));
  float *mine = parts + ((size_t)row * splits + split) * 4;
  mine[0] = r.m;
  mine[1] = r.z;
  mine[2] = r.s;
  __threadfence();
  const int done = atomicAdd(&cnt[row], 1);
  if (done != splits - 1) return;
  __threadfence();
  Tri acc{kNegInf, 0.f, 0.f};
  for (int k = 0; k < splits; k++) {
    const float *q = parts + ((size_t)row * splits + k) * 4;
    Tri o{__hip_atomic_load(q + 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT),
          __hip_atomic_load(q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT),
          __hip_atomic_load(q + 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)};
    acc = tri_merge(acc, o);
  }
  cnt[row] = 0;
  const float H = finish_entropy(acc);
  p.H[row] = H;
  detector_push(p, row, H);
}

}  // namespace

int entropy_splits(int R, int V) {
  // Enough workgroups to cover the chip (~1024), but at least 1024 vectors of
  // 8 logits per workgroup.
  const long nvec = V / 8;
  long s = (1024 + R - 1) / R;
  const long maxs = nvec / 1024 > 0 ? nvec / 1024 : 1;
  if (s > maxs) s = maxs;
  if (s < 1) s = 1;
  if (s > 1024) s = 1024;
  return (int)s;
}

size_t entropy_workspace_bytes(int R, int V) {
  const int s = entropy_splits(R, V);
  if (s == 1) return 0;
  return (((size_t)R * 4 + 15) & ~(size_t)15) + (size_t)R * s * 4 * sizeof(float);
}

hipError_t launch_logit_entropy(const EntropyParams &p, hipStream_t stream) {
  const dim3 grid(p.splits, p.R);
  const size_t esz = p.dtype == 0 ? 4 : 2;
  const bool vec = ((uintptr_t)p.logits % 16 == 0) && ((size_t)p.ld * esz % 16 == 0);
  if (p.dtype == 0) {
    if (vec) hipLaunchKernelGGL((entropy_kernel<float, true>), grid, dim3(kThreads), 0, stream, p);
    else hipLaunchKernelGGL((entropy_kernel<float, false>), grid, dim3(kThreads), 0, stream, p);
  } else {
    if (vec) hipLaunchKernelGGL((entropy_kernel<bf16_t, true>), grid, dim3(kThreads), 0, stream, p);
    else hipLaunchKernelGGL((entropy_kernel<bf16_t, false>), grid, dim3(kThreads), 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace kvr
