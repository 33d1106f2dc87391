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
// workgroup per (sequence, layer, KV head); its waves take 16-row blocks of
// the window rows and make two passes over the keys: the first builds every
// row's softmax maximum and normaliser (online, per lane, then merged across
// the 16 lanes holding the same rows), the second recomputes the logits, forms
// the probabilities and adds their column sums into an LDS accumulator. The
// accumulator is 64-bit fixed point (each column sum rounded to a multiple of
// 2^-32, then added with integer atomics), so the total does not depend on
// the order in which the waves add: the scores are bitwise reproducible. The
// head's scores are written (or added) once at the end, converted back to
// float32. The keys stream through
// an LDS ring shared by the workgroup's eight waves (window_scores_tiled);
// caches too long for the ring beside the accumulator take the older kernel,
// in which each wave of four streams K for its own two row blocks.
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

// Fixed-point column sums of the bf16 kernels: value * 2^32 as int64. A
// column sum is at most G * nq (every window row's whole probability mass),
// far below 2^31, and each addend is rounded once (to 2^-33 at worst).
constexpr double kFix = 4294967296.0;
__device__ __forceinline__ void fix_add(unsigned long long *acc, float v) {
  atomicAdd(acc, (unsigned long long)__double2ll_rn((double)v * kFix));
}
__device__ __forceinline__ float fix_value(unsigned long long a) {
  return (float)((double)(long long)a * (1.0 / kFix));
}

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

template <int D, int NRB>
__device__ __forceinline__ void logits_tile_n(const short4_t (&qa)[NRB][WGeo<D>::KS],
                                              const u32x4 (&kv)[WGeo<D>::NV], float4_t (&c)[NRB]) {
#pragma unroll
  for (int b = 0; b < NRB; b++) c[b] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int t = 0; t < WGeo<D>::KS; t++) {
    const short4_t kb = kstep_op<D>(kv, t);
#pragma unroll
    for (int b = 0; b < NRB; b++) c[b] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(qa[b][t], kb, c[b], 0, 0, 0);
  }
}

template <int D>
__global__ __launch_bounds__(256) void window_scores_bf16(ScoreParams p) {
  extern __shared__ unsigned long long acc[];  // [cap] fixed-point column sums
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
  for (int j = tid; j < n; j += blockDim.x) acc[j] = 0ull;
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
      if (gq == 0 && j < n) fix_add(&acc[j], cs);
    }
  }
  __syncthreads();
  float *sc = p.scores + (size_t)unit * p.cap;
  for (int j = tid; j < n; j += blockDim.x) sc[j] = p.accumulate ? sc[j] + fix_value(acc[j]) : fix_value(acc[j]);
}

// LDS-tiled variant. A workgroup of NW waves holds NW * KRB 16-row blocks of
// the window rows at a time (the A operands in registers) and streams the
// head's keys through a two-tile LDS ring: each tile of kTK keys is brought in
// once per workgroup by buffer-to-LDS loads spread over the waves, then read
// by every wave. K is so read twice (two passes) per group of NW * KRB * 16
// rows, instead of twice per two row blocks per wave. A tile row of D bf16 is
// stored with its 16-byte units swizzled (unit c at c ^ (row mod D/8)), so the
// operand reads (16 keys x one unit each) hit distinct banks. The kernel is
// bound by its arithmetic (two exps per row and key): with NW = 8, KRB = 2
// (4 waves per SIMD) measured fastest, ahead of fewer K passes at KRB = 4.
// The key loads keep the default cache policy: the second pass finds the
// head's keys in L2 (the streaming hint measured 2% slower).
constexpr int kTK = 32;  // keys per LDS tile
constexpr float kSlack = 8.0f;  // log2 units the first pass's reference may trail its maximum

// s_waitcnt vmcnt(n), other counters unconstrained.
template <int N>
__device__ __forceinline__ void wait_vm() {
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

typedef __attribute__((address_space(3))) void lds_void_t;

template <int D, int NW, int KRB>
__global__ __launch_bounds__(NW * 64) void window_scores_tiled(ScoreParams p) {
  constexpr int RU = D / 8;             // 16-byte units per key row
  constexpr int TB = kTK * D * 2;       // bytes per tile
  constexpr int NI = TB / 1024;         // 1 KiB buffer-to-LDS loads per tile
  constexpr int RPI = 1024 / (D * 2);   // key rows per load
  extern __shared__ float smem[];
  unsigned long long *acc = reinterpret_cast<unsigned long long *>(smem);  // [cap] fixed-point column sums
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
  char *ring = reinterpret_cast<char *>(acc + ((p.cap + 1) & ~1));  // [2][TB], 16-byte aligned
  for (int j = tid; j < n; j += NW * kWave) acc[j] = 0ull;
  __syncthreads();

  const int R = p.G * p.nq;
  const bf16_t *Q = static_cast<const bf16_t *>(p.q_win) + (((size_t)s * p.L + l) * p.Hq + (size_t)h * p.G) * p.nq * D;
  const bf16_t *K = static_cast<const bf16_t *>(p.k) + (size_t)unit * p.cap * D;
  const rsrc_t qr = make_rsrc(Q, (uint32_t)R * D * 2u);
  const rsrc_t kr = make_rsrc(K, (uint32_t)n * D * 2u);
  const float c = p.scale * kLog2e;
  const int tiles = (n + kTK - 1) / kTK;
  const int blocks = (R + 15) / 16;
  // This wave's share of a tile's loads: instructions I = wave, wave + NW, ...
  const int mine = (NI - wave + NW - 1) / NW;

  // Tile kt into ring slot kt & 1: load I covers key rows RPI*I .. RPI*I + RPI - 1;
  // lane l writes LDS unit l of the load, which holds key row RPI*I + l / RU,
  // unit (l % RU) ^ (row % RU) of the row.
  auto issue = [&](int kt) {
#if defined(__HIP_DEVICE_COMPILE__)
    char *slot = ring + (kt & 1) * TB;
    for (int I = wave; I < NI; I += NW) {
      const int row = RPI * I + lane / RU;
      const int u = (lane % RU) ^ (row % RU);
      const uint32_t off = ((uint32_t)(kt * kTK + row) * RU + (uint32_t)u) * 16u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(kr, (lds_void_t *)(slot + I * 1024), 16, off, 0, 0, 0);
    }
#else
    (void)kt;  // the host pass has no buffer-to-LDS loads
    (void)kr;
    (void)RPI;
#endif
  };
  // Wait for this wave's loads of the current tile, with `next` of its loads
  // (those of the following tile) allowed to stay in flight.
  auto wait_mine = [&](int next) {
    if (next >= 2) wait_vm<2>();
    else if (next == 1) wait_vm<1>();
    else wait_vm<0>();
  };
  // Operand of 16 keys (subtile st of the tile in `slot`): quarter gq of key
  // row st*16 + col, as kv[NV] 16-byte units.
  auto read_kv = [&](const char *slot, int st, u32x4 (&kv)[WGeo<D>::NV]) {
    const int row = st * 16 + col;
#pragma unroll
    for (int i = 0; i < WGeo<D>::NV; i++) {
      const int u = (gq * WGeo<D>::NV + i) ^ (row % RU);
      kv[i] = *reinterpret_cast<const u32x4 *>(slot + (row * RU + u) * 16);
    }
  };
  // Workgroup barrier without the fence of __syncthreads (whose release
  // would also wait for the next tile's loads in flight): this wave's LDS
  // operations are complete, its tile loads are waited for by wait_mine, and
  // the memory clobber keeps the compiler from moving accesses across it.
  auto bar = [&]() {
    __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));  // lgkmcnt(0)
    asm volatile("s_barrier" ::: "memory");
  };
  // One pass over the keys through the ring; body(kv, key0) per subtile.
  auto stream = [&](auto body) {
    if (tiles > 0) issue(0);
    for (int kt = 0; kt < tiles; kt++) {
      const bool more = kt + 1 < tiles;
      if (more) issue(kt + 1);
      wait_mine(more ? mine : 0);
      bar();  // every wave's loads of tile kt have landed
      const char *slot = ring + (kt & 1) * TB;
#pragma unroll
      for (int st = 0; st < kTK / 16; st++) {
        u32x4 kv[WGeo<D>::NV];
        read_kv(slot, st, kv);
        body(kv, kt * kTK + st * 16);
      }
      bar();  // every wave is done with slot kt & 1 before it is refilled
    }
  };

  for (int g0 = 0; g0 < blocks; g0 += NW * KRB) {
    const int rb = g0 + wave * KRB;
    short4_t qa[KRB][WGeo<D>::KS];
    int nr[KRB][4];
#pragma unroll
    for (int b = 0; b < KRB; b++) {
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
    // Pass 1: per-row maximum and normaliser over the visible keys. The
    // reference m may trail the running maximum by up to kSlack (every term
    // 2^(x - m) stays below 2^kSlack and exact to fp32 rounding), so almost
    // every key costs one exp and no divergent rescale; the merge below
    // settles each row on its true maximum.
    float m[KRB][4], z[KRB][4];
#pragma unroll
    for (int b = 0; b < KRB; b++)
#pragma unroll
      for (int i = 0; i < 4; i++) { m[b][i] = kNegInf; z[b][i] = 0.f; }
    const bool active = rb < blocks;  // wave-uniform: rows of this wave exist
    stream([&](const u32x4 (&kv)[WGeo<D>::NV], int key0) {
      if (!active) return;
      float4_t cc[KRB];
      logits_tile_n<D, KRB>(qa, kv, cc);
      const int j = key0 + col;
      float x[KRB][4];
      bool up = false;
#pragma unroll
      for (int b = 0; b < KRB; b++)
#pragma unroll
        for (int i = 0; i < 4; i++) {
          x[b][i] = j < nr[b][i] ? cc[b][i] * c : kNegInf;
          up |= x[b][i] > m[b][i] + kSlack;
        }
      // The reference moves on the wave's first keys and then rarely: test
      // it for the whole wave, so that the rescale (an exp of its own, which
      // the compiler otherwise issues under a lane mask for every key) is
      // skipped by a uniform branch.
      if (__builtin_amdgcn_ballot_w64(up) != 0) {
#pragma unroll
        for (int b = 0; b < KRB; b++)
#pragma unroll
          for (int i = 0; i < 4; i++)
            if (x[b][i] > m[b][i] + kSlack) {
              z[b][i] = z[b][i] > 0.f ? z[b][i] * fast_exp2(m[b][i] - x[b][i]) : 0.f;
              m[b][i] = x[b][i];
            }
      }
#pragma unroll
      for (int b = 0; b < KRB; b++)
#pragma unroll
        for (int i = 0; i < 4; i++) z[b][i] += fast_exp2(fmaxf(x[b][i] - m[b][i], -256.0f));
    });
    // Merge the 16 lanes that hold the same rows (lane bits 0..3).
#pragma unroll
    for (int msk = 1; msk <= 8; msk <<= 1)
#pragma unroll
      for (int b = 0; b < KRB; b++)
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
#pragma unroll
    for (int b = 0; b < KRB; b++)
#pragma unroll
      for (int i = 0; i < 4; i++) z[b][i] = z[b][i] > 0.f ? 1.0f / z[b][i] : 0.f;  // now 1 / normaliser
    // Pass 2: probabilities, column sums into the LDS accumulator.
    stream([&](const u32x4 (&kv)[WGeo<D>::NV], int key0) {
      if (!active) return;
      float4_t cc[KRB];
      logits_tile_n<D, KRB>(qa, kv, cc);
      const int j = key0 + col;
      float cs = 0.f;
#pragma unroll
      for (int b = 0; b < KRB; b++)
#pragma unroll
        for (int i = 0; i < 4; i++)
          if (j < nr[b][i] && z[b][i] > 0.f) cs += fast_exp2(cc[b][i] * c - m[b][i]) * z[b][i];
      cs += shfl_xor(cs, 16);
      cs += shfl_xor(cs, 32);
      if (gq == 0 && j < n) fix_add(&acc[j], cs);
    });
  }
  __syncthreads();
  float *sc = p.scores + (size_t)unit * p.cap;
  for (int j = tid; j < n; j += NW * kWave) sc[j] = p.accumulate ? sc[j] + fix_value(acc[j]) : fix_value(acc[j]);
}

}  // namespace

size_t window_scores_tiled_lds_bytes(int cap, int D) {
  return ((size_t)((cap + 1) & ~1)) * sizeof(unsigned long long) + 2 * (size_t)kTK * D * 2;
}

hipError_t launch_accumulate_scores(const ScoreParams &p, hipStream_t stream) {
  const dim3 grid(p.S * p.L * p.Hkv);
  if (p.dtype == 0) {
    const size_t lds = ((size_t)p.D + 2 * (size_t)p.cap) * sizeof(float);
    hipLaunchKernelGGL(window_scores_kernel<float>, grid, dim3(64), lds, stream, p);
  } else {
    const size_t tiled = window_scores_tiled_lds_bytes(p.cap, p.D);
    if (tiled <= 65536) {
      if (p.D == 128) hipLaunchKernelGGL((window_scores_tiled<128, 8, 2>), grid, dim3(512), tiled, stream, p);
      else hipLaunchKernelGGL((window_scores_tiled<64, 8, 2>), grid, dim3(512), tiled, stream, p);
    } else {
      // Caches too long for the ring beside the accumulator: one wave streams
      // K per two row blocks (more K traffic, same result).
      const size_t lds = (size_t)p.cap * sizeof(unsigned long long);
      if (p.D == 128) hipLaunchKernelGGL(window_scores_bf16<128>, grid, dim3(256), lds, stream, p);
      else hipLaunchKernelGGL(window_scores_bf16<64>, grid, dim3(256), lds, stream, p);
    }
  }
  return hipGetLastError();
}

}  // namespace kvr
