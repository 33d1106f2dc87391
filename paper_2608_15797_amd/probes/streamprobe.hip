// Memory-access probes for the decode kernels' shapes on gfx950 (measurement
// only; not part of the library). Each probe moves exactly the bytes of the
// kernel it stands for, with that kernel's grid and workgroup shape, and does
// no arithmetic beyond folding the loaded words so the loads are live.
//
//   streamprobe attn N_UNITS CAP N [N ...]
//     Load-only streams of the evicted-cache attention kernel: one 64-lane
//     wave per (sequence, layer, KV head) unit reading the K and V rows of its
//     first N slots (256-byte rows, bf16 D = 128) in chunks of 32 keys, two
//     chunks in flight, 26 KiB of LDS per wave (6 waves per CU), as the kernel.
//     Patterns:
//       mfma  K in the matrix-core operand layout (one load instruction: 64
//             bytes of each of 16 rows), V as four full rows per instruction;
//       rows  K and V both four full rows per instruction;
//       ldsk  K through buffer-to-LDS loads of full rows, V in registers;
//       joint one cache array holding K and V of a slot side by side (512-byte
//             rows), four full K+V rows per two instructions.
//   streamprobe evict N_HEADS CAP B W N
//     The eviction's compaction: one 256-thread workgroup per head, kept rows
//     moved to slots 0..B-1 (the kept set: the first half of the candidates
//     in place, then every other candidate, then the W newest slots), K and V
//     rows of 256 bytes, streaming loads and non-temporal stores. Patterns:
//       inplace  the kernel's chunks: 16 rows read, wait, barrier, written;
//       gather   the same gather into a second array (no hazard, no barrier,
//                all of a head's reads in flight before its writes);
//       copy     a contiguous copy of the same number of bytes per head;
//       flat     one flat streaming copy of the same total bytes, grid-stride.
//   streamprobe read MB [MB ...]
//     Read-only streams of MB megabytes (10^6 bytes), the bound of a call that
//     only reads (the helper's context kernel reads 15032 MB per call of the
//     72B + helper workload). Patterns:
//       flat  grid-stride 16-byte loads, U per thread in flight, 256-thread
//             workgroups, several grid sizes;
//       span  the context kernel's split: one 64-lane wave per equal
//             contiguous span, 1 KiB per load instruction, U in flight, for
//             several wave counts (1024 = one wave per SIMD, as the kernel).
//   streamprobe readpol MB [MB ...]
//     The span pattern through range-checked buffer loads under each cache
//     policy of the load instruction (default, nt, sc0, sc0 nt, sc1, sc1 nt).
//
// Bytes are algorithmic: attention N rows x 512 bytes per unit; eviction the
// moved rows x 512 bytes, read and written.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef __attribute__((address_space(3))) void lds_void_t;

#define CK(x)                                                                      \
  do {                                                                             \
    hipError_t e_ = (x);                                                           \
    if (e_ != hipSuccess) {                                                        \
      printf("HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__);        \
      exit(1);                                                                     \
    }                                                                              \
  } while (0)

constexpr int ROW = 256;       // bytes of one bf16 row at D = 128
constexpr int kStream = 2;     // streaming (nt) cache policy of the buffer loads

__device__ __forceinline__ rsrc_t mk(const void *p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ u32x4 bl(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kStream);
}
__device__ __forceinline__ uint32_t fold(const u32x4 *r, int n) {
  uint32_t a = 0;
  for (int i = 0; i < n; i++) a ^= r[i].x ^ r[i].w;
  return a;
}

// ------------------------------------------------------------ attention loads

// One 32-key chunk of K and V for one lane (c0 = first key).
template <int PAT>
__device__ __forceinline__ void ld_chunk(u32x4 (&k)[8], u32x4 (&v)[8], rsrc_t K, rsrc_t V, int c0, int lane) {
  const int r16 = lane & 15, g4 = lane >> 4;
#pragma unroll
  for (int t = 0; t < 2; t++) {
#pragma unroll
    for (int i = 0; i < 4; i++) {
      if (PAT == 0)  // operand layout: row c0 + 16t + r16, bytes 64 i + 16 g4
        k[4 * t + i] = bl(K, (uint32_t)(c0 + 16 * t + r16) * ROW + i * 64 + g4 * 16);
      else  // four full rows: row c0 + 16t + 4 i + g4, bytes 16 r16
        k[4 * t + i] = bl(K, (uint32_t)(c0 + 16 * t + 4 * i + g4) * ROW + r16 * 16);
    }
#pragma unroll
    for (int c = 0; c < 4; c++) v[4 * t + c] = bl(V, (uint32_t)(c0 + 16 * t + 4 * g4 + c) * ROW + r16 * 16);
  }
}

template <int PAT>
__global__ __launch_bounds__(64) void attn_probe(const char *K, const char *V, int cap, int n, uint32_t *out) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  const int unit = blockIdx.x, lane = threadIdx.x;
  uint32_t acc = 0;
  if (PAT <= 1) {
    const rsrc_t Kr = mk(K + (size_t)unit * cap * ROW, (uint32_t)n * ROW);
    const rsrc_t Vr = mk(V + (size_t)unit * cap * ROW, (uint32_t)n * ROW);
    u32x4 ka[8], va[8], kb[8], vb[8];
    ld_chunk<PAT>(ka, va, Kr, Vr, 0, lane);
    for (int c0 = 0; c0 < n; c0 += 64) {
      ld_chunk<PAT>(kb, vb, Kr, Vr, c0 + 32, lane);
      acc ^= fold(ka, 8) ^ fold(va, 8);
      if (c0 + 32 >= n) break;
      ld_chunk<PAT>(ka, va, Kr, Vr, c0 + 64, lane);
      acc ^= fold(kb, 8) ^ fold(vb, 8);
    }
  } else if (PAT == 2) {
#if defined(__HIP_DEVICE_COMPILE__)
    // K chunks of 32 rows (8 KiB) into a two-slot LDS ring, V in registers.
    const rsrc_t Kr = mk(K + (size_t)unit * cap * ROW, (uint32_t)n * ROW);
    const rsrc_t Vr = mk(V + (size_t)unit * cap * ROW, (uint32_t)n * ROW);
    auto kload = [&](int slot, int c0) {
#pragma unroll
      for (int i = 0; i < 8; i++)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(Kr, (lds_void_t *)(lds + slot * 8192 + i * 1024), 16,
                                                 (uint32_t)(c0 + 4 * i) * ROW + lane * 16, 0, 0, 0);
    };
    auto vload = [&](u32x4 (&v)[8], int c0) {
      const int r16 = lane & 15, g4 = lane >> 4;
#pragma unroll
      for (int t = 0; t < 2; t++)
#pragma unroll
        for (int c = 0; c < 4; c++) v[4 * t + c] = bl(Vr, (uint32_t)(c0 + 16 * t + 4 * g4 + c) * ROW + r16 * 16);
    };
    u32x4 va[8], vb[8];
    kload(0, 0);
    vload(va, 0);
    for (int c0 = 0; c0 < n; c0 += 64) {
      kload(1, c0 + 32);
      vload(vb, c0 + 32);
      // vmcnt(16): the 16 loads of the chunk at c0 + 32 may stay in flight.
      __builtin_amdgcn_s_waitcnt(0 | (7 << 4) | (15 << 8) | (1 << 14));
      acc ^= fold(reinterpret_cast<const u32x4 *>(lds) + lane, 1) ^ fold(va, 8);
      if (c0 + 32 >= n) break;
      kload(0, c0 + 64);
      vload(va, c0 + 64);
      __builtin_amdgcn_s_waitcnt(0 | (7 << 4) | (15 << 8) | (1 << 14));
      acc ^= fold(reinterpret_cast<const u32x4 *>(lds + 8192) + lane, 1) ^ fold(vb, 8);
    }
    __builtin_amdgcn_s_waitcnt(0);  // no buffer-to-LDS load outlives the wave
#endif
  } else {
    // Joint rows: slot j of the unit holds K_j then V_j (512 bytes).
    const rsrc_t R = mk(K + (size_t)unit * cap * 2 * ROW, (uint32_t)n * 2 * ROW);
    const int r16 = lane & 15, g4 = lane >> 4;
    auto ld = [&](u32x4 (&a)[16], int c0) {
#pragma unroll
      for (int i = 0; i < 16; i++)  // 32 slots x 512 bytes = 16 instructions of 1 KiB
        a[i] = bl(R, (uint32_t)(c0 * 2 * ROW) + i * 1024 + (g4 * 16 + r16) * 16);
    };
    u32x4 a[16], b[16];
    ld(a, 0);
    for (int c0 = 0; c0 < n; c0 += 64) {
      ld(b, c0 + 32);
      acc ^= fold(a, 16);
      if (c0 + 32 >= n) break;
      ld(a, c0 + 64);
      acc ^= fold(b, 16);
    }
  }
  out[(size_t)unit * 64 + lane] = acc;
}

// ------------------------------------------------------------ eviction moves

template <int PAT>
__global__ __launch_bounds__(256) void evict_probe(char *K, char *V, char *K2, char *V2, const int *kept, int cap,
                                                   int B) {
  const int head = blockIdx.x, tid = threadIdx.x;
  const size_t hb = (size_t)head * cap * ROW;
  // kept[0..B) is the same for every head; slots before `first` stay.
  __shared__ int first;
  if (tid == 0) {
    int f = B;
    for (int i = 0; i < B; i++)
      if (kept[i] != i) { f = i; break; }
    first = f;
  }
  __syncthreads();
  const int f = first;
  if (PAT == 0) {
    for (int c0 = f; c0 < B; c0 += 16) {
      const int i = c0 + tid / 16, u = tid % 16;
      u32x4 kr = {0, 0, 0, 0}, vr = {0, 0, 0, 0};
      if (i < B) {
        kr = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(K + hb + (size_t)kept[i] * ROW) + u);
        vr = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(V + hb + (size_t)kept[i] * ROW) + u);
      }
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      if (i < B) {
        __builtin_nontemporal_store(kr, reinterpret_cast<u32x4 *>(K + hb + (size_t)i * ROW) + u);
        __builtin_nontemporal_store(vr, reinterpret_cast<u32x4 *>(V + hb + (size_t)i * ROW) + u);
      }
    }
  } else if (PAT == 1 || PAT == 2) {
    // Out of place: up to 8 items per thread in flight (B - f <= 128 rows:
    // 128 rows x 16 units = 2048 items over 256 threads).
    u32x4 kr[8], vr[8];
    const int items = (B - f) * 16;
#pragma unroll
    for (int a = 0; a < 8; a++) {
      const int e = tid + a * 256;
      if (e < items) {
        const int i = f + e / 16, u = e % 16;
        const int src = PAT == 1 ? kept[i] : i;
        kr[a] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(K + hb + (size_t)src * ROW) + u);
        vr[a] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(V + hb + (size_t)src * ROW) + u);
      }
    }
#pragma unroll
    for (int a = 0; a < 8; a++) {
      const int e = tid + a * 256;
      if (e < items) {
        const int i = f + e / 16, u = e % 16;
        __builtin_nontemporal_store(kr[a], reinterpret_cast<u32x4 *>(K2 + hb + (size_t)i * ROW) + u);
        __builtin_nontemporal_store(vr[a], reinterpret_cast<u32x4 *>(V2 + hb + (size_t)i * ROW) + u);
      }
    }
  }
}

__global__ __launch_bounds__(256) void flat_copy(const u32x4 *src, u32x4 *dst, size_t n16) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += (size_t)gridDim.x * 256)
    __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

// ------------------------------------------------------------ read-only streams

template <int U>
__global__ __launch_bounds__(256) void flat_read(const u32x4 *src, size_t n16, uint32_t *out) {
  const size_t stride = (size_t)gridDim.x * 256;
  size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  uint32_t a = 0;
  for (; i + (size_t)(U - 1) * stride < n16; i += (size_t)U * stride) {
    u32x4 r[U];
#pragma unroll
    for (int u = 0; u < U; u++) r[u] = __builtin_nontemporal_load(src + i + (size_t)u * stride);
    a ^= fold(r, U);
  }
  for (; i < n16; i += stride) {
    const u32x4 r = __builtin_nontemporal_load(src + i);
    a ^= r.x ^ r.w;
  }
  out[(size_t)blockIdx.x * 256 + threadIdx.x] = a;
}

template <int U>
__global__ __launch_bounds__(64) void span_read(const u32x4 *src, size_t n16, size_t span16, uint32_t *out) {
  const size_t s0 = (size_t)blockIdx.x * span16;
  const size_t s1 = s0 + span16 < n16 ? s0 + span16 : n16;
  size_t i = s0 + threadIdx.x;
  uint32_t a = 0;
  for (; i + (size_t)(U - 1) * 64 < s1; i += (size_t)U * 64) {
    u32x4 r[U];
#pragma unroll
    for (int u = 0; u < U; u++) r[u] = __builtin_nontemporal_load(src + i + (size_t)u * 64);
    a ^= fold(r, U);
  }
  for (; i < s1; i += 64) {
    const u32x4 r = __builtin_nontemporal_load(src + i);
    a ^= r.x ^ r.w;
  }
  out[(size_t)blockIdx.x * 64 + threadIdx.x] = a;
}

// The span pattern through buffer loads with cache-policy operand AUX (bit 0
// sc0, bit 1 nt, bit 4 sc1): one resource per wave over its span, so every
// load is range-checked.
template <int U, int AUX>
__global__ __launch_bounds__(64) void span_read_pol(const u32x4 *src, size_t n16, size_t span16, uint32_t *out) {
  const size_t s0 = (size_t)blockIdx.x * span16;
  const size_t s1 = s0 + span16 < n16 ? s0 + span16 : n16;
  const uint32_t len = s1 > s0 ? (uint32_t)((s1 - s0) * 16) : 0u;
  const rsrc_t r = mk(src + (s1 > s0 ? s0 : 0), len);
  uint32_t a = 0;
  for (uint32_t off = threadIdx.x * 16u; off < len; off += U * 1024u) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; u++) v[u] = __builtin_amdgcn_raw_buffer_load_b128(r, off + u * 1024u, 0, AUX);
    a ^= fold(v, U);
  }
  out[(size_t)blockIdx.x * 64 + threadIdx.x] = a;
}

template <typename F>
static double time_us(F f, int reps = 20) {
  hipEvent_t a, b;
  CK(hipEventCreate(&a));
  CK(hipEventCreate(&b));
  for (int i = 0; i < 3; i++) f();
  CK(hipGetLastError());
  CK(hipDeviceSynchronize());
  CK(hipEventRecord(a, 0));
  for (int i = 0; i < reps; i++) f();
  CK(hipEventRecord(b, 0));
  CK(hipEventSynchronize(b));
  CK(hipGetLastError());
  float ms = 0;
  CK(hipEventElapsedTime(&ms, a, b));
  CK(hipEventDestroy(a));
  CK(hipEventDestroy(b));
  return ms * 1000.0 / reps;
}

static int run_attn(int units, int cap, const std::vector<int> &ns) {
  const size_t bytes = (size_t)units * cap * ROW;
  char *K, *V, *KV;
  uint32_t *out;
  CK(hipMalloc(&K, bytes));
  CK(hipMalloc(&V, bytes));
  CK(hipMalloc(&KV, 2 * bytes));
  CK(hipMalloc(&out, (size_t)units * 64 * 4));
  CK(hipMemset(K, 1, bytes));
  CK(hipMemset(V, 2, bytes));
  CK(hipMemset(KV, 3, 2 * bytes));
  const size_t lds = 26 * 1024;
  const char *names[4] = {"mfma", "rows", "ldsk", "joint"};
  for (int n : ns) {
    if (n < 1 || n > cap) { printf("n=%d outside 1..cap\n", n); return 1; }
    const double b = (double)units * n * 2 * ROW;
    for (int pat = 0; pat < 4; pat++) {
      double us = time_us([&] {
        switch (pat) {
          case 0: hipLaunchKernelGGL(attn_probe<0>, dim3(units), dim3(64), lds, 0, K, V, cap, n, out); break;
          case 1: hipLaunchKernelGGL(attn_probe<1>, dim3(units), dim3(64), lds, 0, K, V, cap, n, out); break;
          case 2: hipLaunchKernelGGL(attn_probe<2>, dim3(units), dim3(64), lds, 0, K, V, cap, n, out); break;
          default: hipLaunchKernelGGL(attn_probe<3>, dim3(units), dim3(64), lds, 0, KV, V, cap, n, out); break;
        }
      });
      printf("attn units=%d cap=%d n=%d %-6s %9.1f us %6.2f TB/s\n", units, cap, n, names[pat], us, b / (us * 1e-6) / 1e12);
      fflush(stdout);
    }
  }
  CK(hipFree(K)); CK(hipFree(V)); CK(hipFree(KV)); CK(hipFree(out));
  return 0;
}

static int run_evict(int heads, int cap, int B, int W, int n) {
  if (!(0 < W && W < B && B <= n && n <= cap)) { printf("bad evict shape\n"); return 1; }
  // Kept set: candidates [0, n - W); the first half of B - W in place, the
  // rest every other candidate after them, then the W newest slots.
  std::vector<int> kept;
  const int take = B - W, half = take / 2;
  for (int i = 0; i < half; i++) kept.push_back(i);
  for (int j = half + 1; (int)kept.size() < take && j < n - W; j += 2) kept.push_back(j);
  for (int j = half; (int)kept.size() < take; j++) kept.push_back(j);  // (not reached for these shapes)
  for (int w = 0; w < W; w++) kept.push_back(n - W + w);
  int moved = 0;
  for (int i = 0; i < B; i++) {
    if (kept[i] < i || kept[i] >= n || (i && kept[i] <= kept[i - 1])) { printf("bad kept set\n"); return 1; }
    moved += kept[i] != i;
  }
  int f = B;
  for (int i = 0; i < B; i++) if (kept[i] != i) { f = i; break; }
  if ((B - f) * 16 > 2048) { printf("too many moved rows for the gather probe\n"); return 1; }
  const size_t bytes = (size_t)heads * cap * ROW;
  char *K, *V, *K2, *V2;
  int *dk;
  CK(hipMalloc(&K, bytes)); CK(hipMalloc(&V, bytes)); CK(hipMalloc(&K2, bytes)); CK(hipMalloc(&V2, bytes));
  CK(hipMalloc(&dk, B * sizeof(int)));
  CK(hipMemcpy(dk, kept.data(), B * sizeof(int), hipMemcpyHostToDevice));
  CK(hipMemset(K, 1, bytes)); CK(hipMemset(V, 2, bytes));
  const double mb = (double)heads * (B - f) * 2 * ROW * 2;  // rows from the first moved one, read + written
  const double mv = (double)heads * moved * 2 * ROW * 2;
  const char *names[3] = {"inplace", "gather", "copy"};
  for (int pat = 0; pat < 3; pat++) {
    double us = time_us([&] {
      switch (pat) {
        case 0: hipLaunchKernelGGL(evict_probe<0>, dim3(heads), dim3(256), 0, 0, K, V, K2, V2, dk, cap, B); break;
        case 1: hipLaunchKernelGGL(evict_probe<1>, dim3(heads), dim3(256), 0, 0, K, V, K2, V2, dk, cap, B); break;
        default: hipLaunchKernelGGL(evict_probe<2>, dim3(heads), dim3(256), 0, 0, K, V, K2, V2, dk, cap, B); break;
      }
    });
    printf("evict heads=%d cap=%d B=%d W=%d n=%d moved=%d first=%d %-8s %9.1f us %6.2f TB/s (moved rows) %6.2f TB/s (rows from first)\n",
           heads, cap, B, W, n, moved, f, names[pat], us, mv / (us * 1e-6) / 1e12, mb / (us * 1e-6) / 1e12);
    fflush(stdout);
  }
  // Flat copy of the bytes the kernel moves (read + written), one stream.
  const size_t n16 = (size_t)(mb / 2) / 16;
  if (n16 * 16 > bytes) { printf("flat copy too large\n"); return 1; }
  for (int grid : {1024, 2048, 4096}) {
    double us = time_us([&] {
      hipLaunchKernelGGL(flat_copy, dim3(grid), dim3(256), 0, 0, (const u32x4 *)K, (u32x4 *)K2, n16);
    });
    printf("evict flat copy of %zu bytes grid=%d %9.1f us %6.2f TB/s\n", n16 * 16, grid, us, 2.0 * n16 * 16 / (us * 1e-6) / 1e12);
    fflush(stdout);
  }
  CK(hipFree(K)); CK(hipFree(V)); CK(hipFree(K2)); CK(hipFree(V2)); CK(hipFree(dk));
  return 0;
}

static int run_read(const std::vector<double> &mbs) {
  double mx = 0;
  for (double m : mbs) {
    if (!(m >= 1.0 && m <= 64000.0)) { printf("MB=%g outside 1..64000\n", m); return 1; }
    mx = m > mx ? m : mx;
  }
  const size_t cap16 = (size_t)(mx * 1e6) / 16;
  const int grids[4] = {1024, 2048, 4096, 8192};
  const int waves[3] = {1024, 2048, 4096};
  u32x4 *src;
  uint32_t *out;
  CK(hipMalloc(&src, cap16 * 16));
  CK(hipMalloc(&out, (size_t)8192 * 256 * 4));  // the largest grid's threads
  CK(hipMemset(src, 1, cap16 * 16));
  for (double m : mbs) {
    const size_t n16 = (size_t)(m * 1e6) / 16;
    const double b = (double)n16 * 16;
    for (int g : grids) {
      for (int u : {8, 16}) {
        double us = time_us([&] {
          if (u == 8) hipLaunchKernelGGL(flat_read<8>, dim3(g), dim3(256), 0, 0, src, n16, out);
          else hipLaunchKernelGGL(flat_read<16>, dim3(g), dim3(256), 0, 0, src, n16, out);
        });
        printf("read %.0f MB flat grid=%d U=%d %9.1f us %6.2f TB/s\n", m, g, u, us, b / (us * 1e-6) / 1e12);
        fflush(stdout);
      }
    }
    for (int w : waves) {
      const size_t span16 = (n16 + w - 1) / w;
      for (int u : {8, 16}) {
        double us = time_us([&] {
          if (u == 8) hipLaunchKernelGGL(span_read<8>, dim3(w), dim3(64), 0, 0, src, n16, span16, out);
          else hipLaunchKernelGGL(span_read<16>, dim3(w), dim3(64), 0, 0, src, n16, span16, out);
        });
        printf("read %.0f MB span waves=%d U=%d %9.1f us %6.2f TB/s\n", m, w, u, us, b / (us * 1e-6) / 1e12);
        fflush(stdout);
      }
    }
  }
  CK(hipFree(src));
  CK(hipFree(out));
  return 0;
}

// Span reads of MB megabytes under each cache policy of the loads.
static int run_readpol(const std::vector<double> &mbs) {
  double mx = 0;
  for (double m : mbs) {
    if (!(m >= 1.0 && m <= 64000.0)) { printf("MB=%g outside 1..64000\n", m); return 1; }
    mx = m > mx ? m : mx;
  }
  const size_t cap16 = (size_t)(mx * 1e6) / 16;
  u32x4 *src;
  uint32_t *out;
  CK(hipMalloc(&src, cap16 * 16));
  CK(hipMalloc(&out, (size_t)4096 * 64 * 4));
  CK(hipMemset(src, 1, cap16 * 16));
  const char *names[] = {"default", "nt", "sc0", "sc0 nt", "sc1", "sc1 nt"};
  for (double m : mbs) {
    const size_t n16 = (size_t)(m * 1e6) / 16;
    const double b = (double)n16 * 16;
    for (int w : {1024, 2048, 4096}) {
      const size_t span16 = (n16 + w - 1) / w;
      if (span16 * 16 >= (1ull << 31)) { printf("span of %zu bytes exceeds a buffer resource\n", span16 * 16); return 1; }
      for (int pol = 0; pol < 6; pol++) {
        double us = time_us([&] {
          const dim3 g(w), t(64);
          switch (pol) {
            case 0: hipLaunchKernelGGL((span_read_pol<8, 0>), g, t, 0, 0, src, n16, span16, out); break;
            case 1: hipLaunchKernelGGL((span_read_pol<8, 2>), g, t, 0, 0, src, n16, span16, out); break;
            case 2: hipLaunchKernelGGL((span_read_pol<8, 1>), g, t, 0, 0, src, n16, span16, out); break;
            case 3: hipLaunchKernelGGL((span_read_pol<8, 3>), g, t, 0, 0, src, n16, span16, out); break;
            case 4: hipLaunchKernelGGL((span_read_pol<8, 16>), g, t, 0, 0, src, n16, span16, out); break;
            default: hipLaunchKernelGGL((span_read_pol<8, 18>), g, t, 0, 0, src, n16, span16, out); break;
          }
        });
        printf("readpol %.0f MB span waves=%d U=8 policy=%-8s %9.1f us %6.2f TB/s\n", m, w, names[pol], us,
               b / (us * 1e-6) / 1e12);
        fflush(stdout);
      }
    }
  }
  CK(hipFree(src));
  CK(hipFree(out));
  return 0;
}

// Lane layout of the gfx950 lane swaps between 16-lane rows and between
// 32-lane halves: one wave, x = lane id; each lane writes the two results of
// each swap (64 x 4 words). A swap that leaves {l, l^16} (or {l, l^32}) in a
// lane's two results makes their max or sum the xor-16 (xor-32) reduction.
__global__ __launch_bounds__(64) void lane_swap_probe(unsigned *out) {
  const unsigned x = threadIdx.x;
  const auto a = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  const auto b = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  out[threadIdx.x * 4 + 0] = a[0];
  out[threadIdx.x * 4 + 1] = a[1];
  out[threadIdx.x * 4 + 2] = b[0];
  out[threadIdx.x * 4 + 3] = b[1];
}

static int run_lanes() {
  unsigned *d = nullptr, h[256];
  CK(hipMalloc(&d, sizeof(h)));
  hipLaunchKernelGGL(lane_swap_probe, dim3(1), dim3(64), 0, 0, d);
  CK(hipGetLastError());
  CK(hipMemcpy(h, d, sizeof(h), hipMemcpyDeviceToHost));
  CK(hipFree(d));
  bool ok16 = true, ok32 = true;
  for (unsigned l = 0; l < 64; l++) {
    const unsigned p0 = h[4 * l], p1 = h[4 * l + 1], q0 = h[4 * l + 2], q1 = h[4 * l + 3];
    ok16 = ok16 && ((p0 == l && p1 == (l ^ 16)) || (p1 == l && p0 == (l ^ 16)));
    ok32 = ok32 && ((q0 == l && q1 == (l ^ 32)) || (q1 == l && q0 == (l ^ 32)));
    if (l % 8 == 0) printf("lane %2u: swap16 %2u %2u  swap32 %2u %2u\n", l, p0, p1, q0, q1);
  }
  printf("swap16 pairs lane l with l^16: %s\nswap32 pairs lane l with l^32: %s\n", ok16 ? "yes" : "no",
         ok32 ? "yes" : "no");
  return ok16 && ok32 ? 0 : 1;
}

int main(int argc, char **argv) {
  if (argc >= 5 && !strcmp(argv[1], "attn")) {
    std::vector<int> ns;
    for (int i = 4; i < argc; i++) ns.push_back(atoi(argv[i]));
    return run_attn(atoi(argv[2]), atoi(argv[3]), ns);
  }
  if (argc == 7 && !strcmp(argv[1], "evict"))
    return run_evict(atoi(argv[2]), atoi(argv[3]), atoi(argv[4]), atoi(argv[5]), atoi(argv[6]));
  if (argc >= 3 && !strcmp(argv[1], "read")) {
    std::vector<double> mbs;
    for (int i = 2; i < argc; i++) mbs.push_back(atof(argv[i]));
    return run_read(mbs);
  }
  if (argc >= 3 && !strcmp(argv[1], "readpol")) {
    std::vector<double> mbs;
    for (int i = 2; i < argc; i++) mbs.push_back(atof(argv[i]));
    return run_readpol(mbs);
  }
  if (argc == 2 && !strcmp(argv[1], "lanes")) return run_lanes();
  printf("usage: streamprobe attn UNITS CAP N [N ...] | streamprobe evict HEADS CAP B W N | streamprobe read MB [MB ...]"
         " | streamprobe readpol MB [MB ...] | streamprobe lanes\n");
  return 2;
}
