// Full-vocabulary token entropy (Eq. (4)) with the moving-average
// degeneration detector (Sec. 3.2, implementation details), gfx950.
//
// One pass over the logits. Each thread keeps an online triple in the log2
// domain: m = running max of y = inv_temp * x * log2(e), Z = sum 2^(y - m) and
// S = sum (y - m) 2^(y - m), rescaled when m grows. Since the natural-log
// entropy is H = ln Z - (sum (x' - m') e^(x' - m')) / Z with x' the scaled
// logits, in log2 units H = ln2 * (log2 Z - S / Z). Triples merge
// associatively, first across a wave with shuffles, then across the
// workgroup's waves. When a row is split over several workgroups (so that a
// few long rows still fill the chip), each writes its triple to the workspace
// and a second, tiny kernel merges them per row and runs the detector. A
// kernel boundary orders the two: merging inside the first kernel would need
// device-scope fences, which on this chip write back and invalidate the
// per-XCD L2 caches in every workgroup.
//
// Loads are buffer loads from a per-split resource (16 bytes per lane; lanes
// past the split's range return zero without touching memory), issued U at a
// time before any arithmetic, with invalid values masked by selects rather
// than branches.
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

typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ rsrc_t row_rsrc(const void *p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes, 0x00020000);
}

// Vector v (8 logits) of a row through its buffer resource, scaled by c.
__device__ __forceinline__ void load8(rsrc_t r, int v, float c, float (&y)[8], const bf16_t *) {
  const u32x4 w = __builtin_amdgcn_raw_buffer_load_b128(r, (uint32_t)v * 16u, 0, 0);
  y[0] = bf16_lo(w.x) * c; y[1] = bf16_hi(w.x) * c;
  y[2] = bf16_lo(w.y) * c; y[3] = bf16_hi(w.y) * c;
  y[4] = bf16_lo(w.z) * c; y[5] = bf16_hi(w.z) * c;
  y[6] = bf16_lo(w.w) * c; y[7] = bf16_hi(w.w) * c;
}

__device__ __forceinline__ void load8(rsrc_t r, int v, float c, float (&y)[8], const float *) {
  const u32x4 a = __builtin_amdgcn_raw_buffer_load_b128(r, (uint32_t)v * 32u, 0, 0);
  const u32x4 b = __builtin_amdgcn_raw_buffer_load_b128(r, (uint32_t)v * 32u + 16u, 0, 0);
  y[0] = __uint_as_float(a.x) * c; y[1] = __uint_as_float(a.y) * c;
  y[2] = __uint_as_float(a.z) * c; y[3] = __uint_as_float(a.w) * c;
  y[4] = __uint_as_float(b.x) * c; y[5] = __uint_as_float(b.y) * c;
  y[6] = __uint_as_float(b.z) * c; y[7] = __uint_as_float(b.w) * c;
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
    // U vectors of 8 logits per thread per round, all loads issued first.
    constexpr int U = 8;
    const int nvec = p.V / 8;
    const int per = (nvec + splits - 1) / splits;
    const int v0 = split * per;
    const int v1 = min(v0 + per, nvec);
    // The resource ends where this split's vectors end, so the lanes of a
    // partly used round load nothing instead of fetching the next split.
    const rsrc_t rr = row_rsrc(x, (uint32_t)v1 * 8u * (uint32_t)sizeof(T));
    for (int base = v0 + tid; base < v1; base += U * kThreads) {
      float y[U][8];
#pragma unroll
      for (int u = 0; u < U; u++) load8(rr, base + u * kThreads, c, y[u], x);
#pragma unroll
      for (int u = 0; u < U; u++) {
        const bool ok = base + u * kThreads < v1;
#pragma unroll
        for (int e = 0; e < 8; e++) y[u][e] = ok ? y[u][e] : kNegInf;
      }
      float lm = kNegInf;
#pragma unroll
      for (int u = 0; u < U; u++)
#pragma unroll
        for (int e = 0; e < 8; e++) lm = fmaxf(lm, y[u][e]);
      if (lm > t.m) {
        if (t.z > 0.f) {
          const float f = fast_exp2(t.m - lm);
          t.s = (t.s + (t.m - lm) * t.z) * f;
          t.z *= f;
        }
        t.m = lm;
      }
#pragma unroll
      for (int u = 0; u < U; u++)
#pragma unroll
        for (int e = 0; e < 8; e++) {
          const float d = fmaxf(y[u][e] - t.m, -256.0f);
          const float w = fast_exp2(d);
          t.z += w;
          t.s = fmaf(d, w, t.s);
        }
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
  float *mine = static_cast<float *>(p.ws) + ((size_t)row * splits + split) * 4;
  mine[0] = r.m;
  mine[1] = r.z;
  mine[2] = r.s;
}

// Per-row merge of the split partials, then the detector; one thread per row.
__global__ __launch_bounds__(256) void entropy_merge(EntropyParams p) {
  const int row = blockIdx.x * blockDim.x + threadIdx.x;
  if (row >= p.R) return;
  const float *q = static_cast<const float *>(p.ws) + (size_t)row * p.splits * 4;
  Tri acc{kNegInf, 0.f, 0.f};
  for (int k = 0; k < p.splits; k++) acc = tri_merge(acc, Tri{q[4 * k], q[4 * k + 1], q[4 * k + 2]});
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
  return (size_t)R * s * 4 * sizeof(float);
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
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.splits == 1) return e;
  hipLaunchKernelGGL(entropy_merge, dim3((p.R + 255) / 256), dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace kvr
