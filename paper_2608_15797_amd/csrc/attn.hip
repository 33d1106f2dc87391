// Grouped-query decode attention for KV-Rescue candidate batches on gfx950.
//
// Computes, per candidate s, layer l and query head qh (KV head h = qh / G),
// o = sum_j softmax_j(scale * q.k_j) v_j over the sequence's live cache
// entries (Eq. (1), third line), optionally preceded by a shared full-context
// prefix (the helper of Sec. 3.1), and streams the per-KV-head attention mass
// that forms the accumulated-attention importance score (Sec. 2.1).
//
// bf16 path: one 64-lane wave per (sequence, layer, KV head) unit. The G query
// heads of a KV head form the 16 rows of an MFMA tile, so q.K^T and P.V are
// 16x16x16 bf16 matrix-core products:
//   * S^T = K . Q^T : A = 16 keys x 16 d (each lane loads 16 contiguous bytes of
//     one key row), B = Q^T held in registers for the whole unit. The output
//     layout (lane = query row + 16 * key group) is exactly the A-operand
//     layout P needs for P . V, so probabilities never leave registers.
//   * O = P . V : B = 16 keys x 16 d. Each lane loads 16 contiguous bytes of
//     four consecutive key rows (fully coalesced: 4 rows x 256 B per load
//     instruction) and transposes 4x8 bf16 in registers with bit operations,
//     which assigns output column n to d = n * (D/16) + b for instance b.
// Keys stream in chunks of 32 through buffer loads (wave-uniform base and
// range in SGPRs, 32-bit lane offsets, zero fill past the range), double
// buffered so one chunk's loads are in flight while the previous one is
// computed. The softmax is online with running max and sum kept in the log2
// domain. Logits of window steps go to LDS so the normalised probabilities
// can be summed over the G heads after the last chunk.
//
// Helper (prefix) path: split-K over the prefix. Each wave processes the query
// rows of all candidates sharing a prefix (up to 4 row blocks = 64 rows), so
// shared context is read from HBM once per step, and writes (max, sum,
// unnormalised o) partials. The waves are exactly as many as fit on the chip
// at once, each taking an equal span of the flattened (prefix, layer, KV
// head, key) space (one partial per unit its span touches), so all of them
// finish in one round. The private suffix then runs as its own unit per
// (candidate, layer, KV head) and folds those partials in by log-sum-exp.
//
// f32 path: plain VALU kernel (one wave per unit) for float32 caches.
//
// This file is compiled twice. With KVR_ATTN_WIDE = 1 (attn_wide.hip) it
// provides only the context kernels of three and four row blocks
// (launch_prefix_wide, prefix_slots_wide), built with the matrix-core
// accumulators in vector registers; every other kernel and entry point comes
// from the KVR_ATTN_WIDE = 0 build.
#include <hip/hip_runtime.h>

#include <atomic>

#include "entropy_common.h"
#include "sampler_common.h"
#include "kvr_device.h"
#include "kvr_internal.h"

#ifndef KVR_ATTN_WIDE
#define KVR_ATTN_WIDE 0
#endif

namespace kvr {

namespace {


template <int D>
struct Geo {
  static constexpr int NB = D / 16;   // MFMA instances per 16-key tile
  static constexpr int NLD = D / 32;  // 16-byte loads per lane per K row
  static constexpr int VW = NB / 2;   // 32-bit words per lane per V row
};

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// A split-K partial record of one query row: (max, sum, -, -) as float32 in
// the log2 domain, then o / sum as D float16 (the sum-normalised output, at
// most max |v| in size), so 4 + D/2 float slots, a multiple of 16 bytes.
template <int D>
constexpr int kRecFloats = 4 + D / 2;

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef float f32x2v_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pack_f16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2v_t){a, b}, half2_t));
}
__device__ __forceinline__ float f16_lo(uint32_t w) { return (float)__builtin_bit_cast(half2_t, w)[0]; }
__device__ __forceinline__ float f16_hi(uint32_t w) { return (float)__builtin_bit_cast(half2_t, w)[1]; }

__device__ __forceinline__ short4_t s4(uint32_t a, uint32_t b) {
  u32x2 v = {a, b};
  return __builtin_bit_cast(short4_t, v);
}

__device__ __forceinline__ float4_t mfma16(short4_t a, short4_t b, float4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}

// Q^T operands of one query row (or zeros). d(g, b, c) = (b/2)*32 + g*8 + (b%2)*4 + c.
template <int D>
__device__ __forceinline__ void load_qop(const bf16_t *qrow, int g4, short4_t (&qop)[Geo<D>::NB]) {
#pragma unroll
  for (int i = 0; i < Geo<D>::NLD; i++) {
    u32x4 w = {0u, 0u, 0u, 0u};
    if (qrow) w = *reinterpret_cast<const u32x4 *>(qrow + i * 32 + g4 * 8);
    qop[2 * i] = s4(w.x, w.y);
    qop[2 * i + 1] = s4(w.z, w.w);
  }
}

// Buffer resources: a wave-uniform base address and byte range in SGPRs, so
// per-lane addressing is a 32-bit offset and loads past the range return 0.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef __attribute__((address_space(3))) void lds_void_t;

// s_waitcnt vmcnt(0), other counters unconstrained.
__device__ __forceinline__ void wait_vm0() { __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8)); }

__device__ __forceinline__ rsrc_t make_rsrc(const void *p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes, 0x00020000);
}

// K and V data of one chunk of TILES*16 keys, as loaded by one lane:
// k[t][i]: 16 bytes of key row c0 + 16t + (lane & 15) at d = 32i + 8*(lane >> 4);
// v[t][c]: D/16 elements of value row c0 + 16t + 4*(lane >> 4) + c at d = (lane & 15) * D/16.
template <int D, int TILES>
struct KVChunk {
  u32x4 k[TILES][Geo<D>::NLD];
  uint32_t v[TILES][4][Geo<D>::VW];
};

template <int D, int TILES>
__device__ __forceinline__ void load_chunk(KVChunk<D, TILES> &c, rsrc_t K, rsrc_t V, int c0,
                                           int r16, int g4) {
  constexpr uint32_t ROW = D * 2;
#pragma unroll
  for (int t = 0; t < TILES; t++) {
    const uint32_t base = (uint32_t)(c0 + t * 16 + r16) * ROW + g4 * 16;
#pragma unroll
    for (int i = 0; i < Geo<D>::NLD; i++)
      c.k[t][i] = __builtin_amdgcn_raw_buffer_load_b128(K, base + i * 64, 0, kStreamLoad);
  }
#pragma unroll
  for (int t = 0; t < TILES; t++)
#pragma unroll
    for (int cc = 0; cc < 4; cc++) {
      const uint32_t off = (uint32_t)(c0 + t * 16 + 4 * g4 + cc) * ROW + r16 * (Geo<D>::NB * 2);
      if constexpr (D == 128) {
        const u32x4 x = __builtin_amdgcn_raw_buffer_load_b128(V, off, 0, kStreamLoad);
        c.v[t][cc][0] = x.x; c.v[t][cc][1] = x.y; c.v[t][cc][2] = x.z; c.v[t][cc][3] = x.w;
      } else {
        const u32x2 x = __builtin_amdgcn_raw_buffer_load_b64(V, off, 0, kStreamLoad);
        c.v[t][cc][0] = x.x; c.v[t][cc][1] = x.y;
      }
    }
}

// Logits (log2 domain) of one chunk for one 16-row block: S^T = K . Q^T.
// Only a tail chunk (wave-uniform flag) can hold keys at or beyond nlim;
// those are masked to -inf.
template <int D, int TILES>
__device__ __forceinline__ void chunk_logits(const KVChunk<D, TILES> &c, const short4_t (&qop)[Geo<D>::NB],
                                             float (&x)[TILES][4], int c0, int nlim, int g4, float sl2,
                                             bool tail) {
#pragma unroll
  for (int t = 0; t < TILES; t++) {
    float4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < Geo<D>::NLD; i++) {
      acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(s4(c.k[t][i].x, c.k[t][i].y), qop[2 * i], acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(s4(c.k[t][i].z, c.k[t][i].w), qop[2 * i + 1], acc, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 4; i++) x[t][i] = acc[i] * sl2;
    if (tail) {
#pragma unroll
      for (int i = 0; i < 4; i++) {
        const int key = c0 + t * 16 + 4 * g4 + i;
        x[t][i] = key < nlim ? x[t][i] : kNegInf;
      }
    }
  }
}

// Stream chunks of CH = 16*TILES keys over [k0, k1) through a DEPTH-deep ring
// of register buffers: DEPTH-1 chunks are in flight while one is processed.
// Loads past the resource's range return zero without touching memory, so
// the ring is refilled unconditionally; pre() runs once the first loads are
// in flight, then proc(chunk, c0) sees each real chunk.
// stream_chunks with the ring supplied by the caller, whose buf[0] already
// holds (or is loading) the chunk at k0.
template <int D, int TILES, int DEPTH, typename Pre, typename Proc>
__device__ __forceinline__ void stream_chunks_from(KVChunk<D, TILES> (&buf)[DEPTH], rsrc_t K, rsrc_t V, int k0,
                                                   int k1, int r16, int g4, Pre pre, Proc proc) {
  constexpr int stride = 16 * TILES;
#pragma unroll
  for (int s = 1; s < DEPTH - 1; s++) load_chunk<D, TILES>(buf[s], K, V, k0 + s * stride, r16, g4);
  pre();
  for (int c0 = k0; c0 < k1; c0 += DEPTH * stride) {
#pragma unroll
    for (int j = 0; j < DEPTH; j++) {
      const int cj = c0 + j * stride;
      if (cj >= k1) break;
      load_chunk<D, TILES>(buf[(j + DEPTH - 1) % DEPTH], K, V, cj + (DEPTH - 1) * stride, r16, g4);
      proc(buf[j], cj);
    }
  }
}

template <int D, int TILES, int DEPTH, typename Pre, typename Proc>
__device__ __forceinline__ void stream_chunks(rsrc_t K, rsrc_t V, int k0, int k1, int r16, int g4,
                                              Pre pre, Proc proc) {
  constexpr int stride = 16 * TILES;
  KVChunk<D, TILES> buf[DEPTH];
#pragma unroll
  for (int s = 0; s < DEPTH - 1; s++) load_chunk<D, TILES>(buf[s], K, V, k0 + s * stride, r16, g4);
  pre();
  for (int c0 = k0; c0 < k1; c0 += DEPTH * stride) {
#pragma unroll
    for (int j = 0; j < DEPTH; j++) {
      const int cj = c0 + j * stride;
      if (cj >= k1) break;
      load_chunk<D, TILES>(buf[(j + DEPTH - 1) % DEPTH], K, V, cj + (DEPTH - 1) * stride, r16, g4);
      proc(buf[j], cj);
    }
  }
}

// s_waitcnt vmcnt(N), other counters unconstrained (N < 64).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Evicted-cache chunks with the key rows in LDS: key rows are read as whole
// rows (four 256-byte rows per 1 KiB instruction at D = 128) by buffer-to-LDS
// loads into a ring slot, and the matrix-core operands are read back from
// there. Loading the operand layout directly would take 64 bytes of each of 16
// rows per instruction, which streams measurably slower from HBM. The 16-byte
// units of a row are stored rotated by the row index (unit u of row r at
// position u ^ (r mod units per row)), so the 16 lanes reading one unit of 16
// consecutive rows hit distinct banks. Value rows stay in registers.
template <int D>
struct KLds {
  static constexpr int ROW = D * 2;        // bytes per key row
  static constexpr int RU = ROW / 16;      // 16-byte units per row
  static constexpr int RPI = 1024 / ROW;   // rows per buffer-to-LDS instruction
};

template <int D, int TILES>
struct VChunk {
  uint32_t v[TILES][4][Geo<D>::VW];
};

// Per-lane byte offsets of the loads of one chunk, relative to the chunk's
// first row; they do not change from chunk to chunk (the chunk's base goes
// into the buffer resource), so the stream loop does no vector address
// arithmetic. Key load I covers rows RPI*I .. RPI*I + RPI - 1: lane l writes
// LDS unit l of the load, which holds row RPI*I + l / RU, unit
// (l % RU) ^ (row % RU). Value loads: row 16t + 4 g4 + cc at byte 16 r16 *
// (D / 128), the cc rows apart by ROW bytes (the instruction offset).
template <int D, int TILES>
struct KLOffsets {
  static constexpr int KI = 16 * TILES * KLds<D>::ROW / 1024;
  uint32_t k[KI];
  uint32_t v[TILES];
  __device__ __forceinline__ explicit KLOffsets(int lane) {
#pragma unroll
    for (int I = 0; I < KI; I++) {
      const int row = KLds<D>::RPI * I + lane / KLds<D>::RU;
      const int u = (lane % KLds<D>::RU) ^ (row % KLds<D>::RU);
      k[I] = (uint32_t)row * KLds<D>::ROW + (uint32_t)u * 16u;
    }
    const int r16 = lane & 15, g4 = lane >> 4;
#pragma unroll
    for (int t = 0; t < TILES; t++) v[t] = (uint32_t)(t * 16 + 4 * g4) * (D * 2) + (uint32_t)r16 * (Geo<D>::NB * 2);
  }
};

// Loads of one chunk of 16*TILES keys starting at row c0 of the unit's K and
// V (kbase, vbase) with `rows` rows readable from kbase/vbase (loads past them
// return zero): the key rows into `slot` (LDS), then the value rows into
// registers. Issues KI + 4 * TILES vector-memory instructions.
template <int D, int TILES>
__device__ __forceinline__ void load_chunk_lds(VChunk<D, TILES> &c, char *slot, const bf16_t *kbase, const bf16_t *vbase,
                                               int rows, int c0, const KLOffsets<D, TILES> &off) {
  constexpr uint32_t ROW = D * 2;
  const uint32_t bytes = rows > c0 ? (uint32_t)(rows - c0) * ROW : 0u;
  const rsrc_t K = make_rsrc(kbase + (size_t)c0 * D, bytes);
  const rsrc_t V = make_rsrc(vbase + (size_t)c0 * D, bytes);
#if defined(__HIP_DEVICE_COMPILE__)
#pragma unroll
  for (int I = 0; I < KLOffsets<D, TILES>::KI; I++)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(K, (lds_void_t *)(slot + I * 1024), 16, off.k[I], 0, 0, 0);
#else
  (void)K;  // the host pass has no buffer-to-LDS loads
#endif
#pragma unroll
  for (int t = 0; t < TILES; t++)
#pragma unroll
    for (int cc = 0; cc < 4; cc++) {
      if constexpr (D == 128) {
        const u32x4 x = __builtin_amdgcn_raw_buffer_load_b128(V, off.v[t] + cc * ROW, 0, kStreamLoad);
        c.v[t][cc][0] = x.x; c.v[t][cc][1] = x.y; c.v[t][cc][2] = x.z; c.v[t][cc][3] = x.w;
      } else {
        const u32x2 x = __builtin_amdgcn_raw_buffer_load_b64(V, off.v[t] + cc * ROW, 0, kStreamLoad);
        c.v[t][cc][0] = x.x; c.v[t][cc][1] = x.y;
      }
    }
}

// Logits (log2 domain) of one LDS-resident chunk for one 16-row block, as
// chunk_logits: key row 16t + r16, operand unit 4i + g4 (d = 32i + 8 g4).
template <int D, int TILES>
__device__ __forceinline__ void chunk_logits_lds(const char *slot, const short4_t (&qop)[Geo<D>::NB],
                                                 float (&x)[TILES][4], int c0, int nlim, int r16, int g4,
                                                 float sl2, bool tail) {
#pragma unroll
  for (int t = 0; t < TILES; t++) {
    const int row = t * 16 + r16;
    float4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < Geo<D>::NLD; i++) {
      const int u = (4 * i + g4) ^ (row % KLds<D>::RU);
      const u32x4 kk = *reinterpret_cast<const u32x4 *>(slot + row * KLds<D>::ROW + u * 16);
      acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(s4(kk.x, kk.y), qop[2 * i], acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(s4(kk.z, kk.w), qop[2 * i + 1], acc, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 4; i++) x[t][i] = acc[i] * sl2;
    if (tail) {
#pragma unroll
      for (int i = 0; i < 4; i++) {
        const int key = c0 + t * 16 + 4 * g4 + i;
        x[t][i] = key < nlim ? x[t][i] : kNegInf;
      }
    }
  }
}

// stream_chunks_from for LDS-resident key rows: chunk c (from k0) sits in
// ring slot c % DEPTH (slots of 16*TILES*2D bytes from `ring`) and value
// register buffer c % DEPTH; buffer 0 / slot 0 already hold (or are loading)
// the chunk at k0. Keys [k0, k1) of kbase / vbase are read. Before a chunk is
// processed the wave waits until only the loads of the chunks after it are in
// flight: nothing else is issued inside the loop, so that count is exact.
template <int D, int TILES, int DEPTH, typename Pre, typename Proc>
__device__ __forceinline__ void stream_chunks_lds(VChunk<D, TILES> (&buf)[DEPTH], char *ring, const bf16_t *kbase,
                                                  const bf16_t *vbase, int k0, int k1,
                                                  const KLOffsets<D, TILES> &off, Pre pre, Proc proc) {
  constexpr int stride = 16 * TILES;
  constexpr int SLOT = 16 * TILES * KLds<D>::ROW;
  constexpr int PER = KLOffsets<D, TILES>::KI + 4 * TILES;  // instructions per chunk
#pragma unroll
  for (int s = 1; s < DEPTH - 1; s++)
    load_chunk_lds<D, TILES>(buf[s], ring + s * SLOT, kbase, vbase, k1, k0 + s * stride, off);
  pre();
  for (int c0 = k0; c0 < k1; c0 += DEPTH * stride) {
#pragma unroll
    for (int j = 0; j < DEPTH; j++) {
      const int cj = c0 + j * stride;
      if (cj >= k1) break;
      const int nb = (j + DEPTH - 1) % DEPTH;
      load_chunk_lds<D, TILES>(buf[nb], ring + nb * SLOT, kbase, vbase, k1, cj + (DEPTH - 1) * stride, off);
      wait_vm<PER * (DEPTH - 1)>();
      proc(buf[j], ring + j * SLOT, cj);
    }
  }
}

// B operands of P.V for every instance b of every tile, from the four V rows
// (keys 4*g4 + c, c = 0..3) each lane holds: operand b packs element b of
// the four rows. Built once per chunk and shared by all row blocks.
template <int D, int TILES>
__device__ __forceinline__ void make_vops(const uint32_t (&v)[TILES][4][Geo<D>::VW],
                                          short4_t (&vo)[TILES][Geo<D>::NB]) {
#pragma unroll
  for (int t = 0; t < TILES; t++)
#pragma unroll
    for (int w = 0; w < Geo<D>::VW; w++) {
      vo[t][2 * w] = s4(__builtin_amdgcn_perm(v[t][1][w], v[t][0][w], 0x05040100u),
                        __builtin_amdgcn_perm(v[t][3][w], v[t][2][w], 0x05040100u));
      vo[t][2 * w + 1] = s4(__builtin_amdgcn_perm(v[t][1][w], v[t][0][w], 0x07060302u),
                            __builtin_amdgcn_perm(v[t][3][w], v[t][2][w], 0x07060302u));
    }
}

// Operand b of one tile, built on the fly (single-row-block kernels).
template <int D>
__device__ __forceinline__ short4_t make_vop(const uint32_t (&v)[4][Geo<D>::VW], int b) {
  const int w = b >> 1;
  const uint32_t sel = (b & 1) ? 0x07060302u : 0x05040100u;
  return s4(__builtin_amdgcn_perm(v[1][w], v[0][w], sel), __builtin_amdgcn_perm(v[3][w], v[2][w], sel));
}

typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Four probabilities -> A operand of P.V (hardware round-to-nearest-even).
__device__ __forceinline__ short4_t pop4(float a, float b, float c, float d) {
  const bf16x2_t lo = __builtin_convertvector((f32x2_t){a, b}, bf16x2_t);
  const bf16x2_t hi = __builtin_convertvector((f32x2_t){c, d}, bf16x2_t);
  return s4(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
}

// Online-softmax state of the lane's query row within one 16-row block.
struct RowState {
  float m;   // running max of logits (log2 domain)
  float zl;  // lane-local partial sum of exp2(x - m)
};

// Process one chunk of TILES*16 keys for one row block. x[t][i] are the
// lane's logits (log2 domain, masked = -inf). Updates state, rescales o and
// accumulates P.V with the chunk's V rows.
template <int D, int TILES, bool LAZY, typename VOp>
__device__ __forceinline__ void softmax_pv_core(float (&x)[TILES][4], RowState &st,
                                                float4_t (&o)[Geo<D>::NB], VOp vop, int g4) {
  float cm = kNegInf;
#pragma unroll
  for (int t = 0; t < TILES; t++)
#pragma unroll
    for (int i = 0; i < 4; i++) cm = fmaxf(cm, x[t][i]);
  cm = fmaxf(cm, shfl_xor(cm, 16));
  cm = fmaxf(cm, shfl_xor(cm, 32));
  // LAZY: the reference st.m may trail the row's running
  // maximum by up to kLagLog2 (probabilities up to 2^kLagLog2 before the
  // normalisation, exact in float32 and bf16 alike), and moves only when a
  // chunk exceeds it by more; the rescale of o then runs only on those rare
  // chunks. With many rows per tile some row's maximum grows in most chunks,
  // so the exact update rescaled (and moved the accumulators through VALU)
  // almost every chunk. Otherwise the reference is the running maximum.
  constexpr float kLagLog2 = 8.0f;
  const bool need = LAZY ? cm > st.m + kLagLog2 : cm > st.m;
  const float mn = need ? cm : st.m;
  const bool live = mn != kNegInf;
  const float alpha = live ? fast_exp2(st.m - mn) : 1.0f;
  float psum = 0.0f;
#pragma unroll
  for (int t = 0; t < TILES; t++)
#pragma unroll
    for (int i = 0; i < 4; i++) {
      x[t][i] = live ? fast_exp2(x[t][i] - mn) : 0.0f;
      psum += x[t][i];
    }
  st.zl = st.zl * alpha + psum;
  const bool grew = need;
  st.m = mn;
  // o rows are 4*g4 + i; their alphas live in lanes 4*g4 + i.
  if (!LAZY || __any(grew)) {
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const float ai = __shfl(alpha, 4 * g4 + i, kWave);
#pragma unroll
      for (int b = 0; b < Geo<D>::NB; b++) o[b][i] *= ai;
    }
  }
#pragma unroll
  for (int t = 0; t < TILES; t++) {
    const short4_t pa = pop4(x[t][0], x[t][1], x[t][2], x[t][3]);
#pragma unroll
    for (int b = 0; b < Geo<D>::NB; b++) o[b] = mfma16(pa, vop(t, b), o[b]);
  }
}

// With V operands prebuilt by make_vops (shared by several row blocks).
template <int D, int TILES, bool LAZY = false>
__device__ __forceinline__ void softmax_pv(float (&x)[TILES][4], RowState &st, float4_t (&o)[Geo<D>::NB],
                                           const short4_t (&vo)[TILES][Geo<D>::NB], int g4) {
  softmax_pv_core<D, TILES, LAZY>(x, st, o, [&](int t, int b) { return vo[t][b]; }, g4);
}

// With V operands built on the fly from the raw rows.
template <int D, int TILES, bool LAZY = false>
__device__ __forceinline__ void softmax_pv(float (&x)[TILES][4], RowState &st, float4_t (&o)[Geo<D>::NB],
                                           const uint32_t (&v)[TILES][4][Geo<D>::VW], int g4) {
  softmax_pv_core<D, TILES, LAZY>(x, st, o, [&](int t, int b) { return make_vop<D>(v[t], b); }, g4);
}

// ---------------------------------------------------------------------------
// Own-cache kernel: base (evicted cache, optional score streaming) or helper
// suffix (MERGE: runs after the context kernel on the same stream and folds
// that kernel's split partials of its rows into its own softmax state before
// writing the output, so no separate merge pass is needed).
// Keys [0, n-1) stream from the cache in chunks of 32, double-buffered so the
// next chunk's loads are in flight while the current one is computed; the
// appended token (slot n-1) is a final one-key tile read from k_new/v_new.
constexpr size_t kBaseLdsFloor = 26 * 1024;  // see the evicted-cache launch
constexpr size_t kMaxLds = 64 * 1024;        // LDS a workgroup may ask for
constexpr int kFastPieces = 4;  // split partials per row merged with batched LDS reads
constexpr size_t kMergePrefetchBytes = 16384;  // LDS for the suffix kernel's prefetched partials
constexpr bool kSuffixKl = true;               // suffix kernel with its key rows through the LDS ring

// KL (evicted cache only): key rows through an LDS ring (load_chunk_lds)
// instead of registers; the ring takes the first kl_ring<D, TILES, DEPTH>
// bytes of LDS.
template <int D, int TILES, int DEPTH>
constexpr size_t kl_ring = (size_t)DEPTH * 16 * TILES * D * 2;
// Chunk shape of the evicted-cache launch with LDS key rows.
constexpr int kKlTiles = 2;
constexpr int kKlDepth = 2;

// LT (evicted cache only): 0, or the logit type of the step's entropy rows
// computed in the same launch (1 = bfloat16, 2 = float32; 3 and 4 the same
// with the sampler). The first e.row0[e.nsets] workgroups of the grid are
// then one wave per logit row (entropy_row_wave: the whole row, its entropy
// and detector update, no partials; entropy_sample_row_wave also draws the
// row's next token from its k best logits, using the launch's LDS for the
// candidates); they are dispatched first and stream their rows while the
// attention units run. The other workgroups are the attention units.
template <int D, bool MERGE, int TILES, int DEPTH, bool KL = false, int LT = 0>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(2))) void attn_cache_bf16(AttnParams p,
                                                                                               EntropyBatch e) {
  static_assert(!(LT && MERGE), "entropy rows ride with the evicted cache");
  constexpr int CH = 16 * TILES;
  constexpr int NB = Geo<D>::NB;
  constexpr uint32_t ROW = D * 2;
  extern __shared__ float smem[];

  int unit = blockIdx.x;  // ((s * L) + l) * Hkv + h
  if constexpr (LT != 0) {
    const int rows = e.row0[e.nsets];
    if (unit < rows) {
      const int k = batch_set(e, unit);
      uint64_t *cand = reinterpret_cast<uint64_t *>(smem);
      if constexpr (LT == 1)
        entropy_row_wave<bf16_t, 12>(e.set[k], unit - e.row0[k], threadIdx.x);
      else if constexpr (LT == 2)
        entropy_row_wave<float, 6>(e.set[k], unit - e.row0[k], threadIdx.x);
      else if constexpr (LT == 3)
        entropy_sample_row_wave<bf16_t, 8>(e.set[k], unit - e.row0[k], threadIdx.x, cand);
      else
        entropy_sample_row_wave<float, 4>(e.set[k], unit - e.row0[k], threadIdx.x, cand);
      return;
    }
    unit -= rows;
  }
  const int h = unit % p.Hkv;
  const int sl = unit / p.Hkv;
  const int l = sl % p.L;
  const int s = sl / p.L;
  const int lane = threadIdx.x;
  const int r16 = lane & 15;
  const int g4 = lane >> 4;
  const int G = p.G;
  const int qh0 = h * G;
  const size_t qrow0 = ((size_t)s * p.L + l) * p.Hq + qh0;
  const size_t ubase = (size_t)unit * p.cap * D;
  bf16_t *Kc = static_cast<bf16_t *>(p.k) + ubase;
  bf16_t *Vc = static_cast<bf16_t *>(p.v) + ubase;
  const bf16_t *kn = p.k_new ? static_cast<const bf16_t *>(p.k_new) + (size_t)unit * D : nullptr;
  const bf16_t *vn = p.v_new ? static_cast<const bf16_t *>(p.v_new) + (size_t)unit * D : nullptr;

  // The loads that do not depend on the live length are issued before it is
  // read: the query rows and the new token's one-key tile and, for an evicted
  // cache (whose live length is at least B once the prompt is in), the first
  // cache chunk, read over the first min(cap, CH) slots. A unit then exposes
  // one memory round trip instead of two. Slots of that chunk at or past the
  // end of the live cache hold stale rows: their keys are masked to -inf like
  // any tail chunk's, and their value rows are zeroed before use (a stale row
  // may hold NaN, and 0 * NaN would reach the output). A suffix cache starts
  // empty after every committed step, so there the chunk waits for the length
  // and reads no stale rows.
  short4_t qop[NB];
  load_qop<D>(r16 < G ? static_cast<const bf16_t *>(p.q) + (qrow0 + r16) * D : nullptr, g4, qop);
  KVChunk<D, 1> cn;
  if (kn) load_chunk<D, 1>(cn, make_rsrc(kn, ROW), make_rsrc(vn, ROW), 0, r16, g4);
  KVChunk<D, TILES> ring[KL ? 1 : DEPTH];
  VChunk<D, TILES> vring[KL ? DEPTH : 1];
  char *kring = reinterpret_cast<char *>(smem);  // KL: [DEPTH][CH rows of ROW bytes]
  float *pbuf = smem + (KL ? kl_ring<D, TILES, DEPTH> / sizeof(float) : 0);  // MERGE: prefetched partials
  const KLOffsets<D, TILES> kloff(lane);
  if constexpr (!MERGE) {
    const int first = p.cap < CH ? p.cap : CH;
    if constexpr (KL)
      load_chunk_lds<D, TILES>(vring[0], kring, Kc, Vc, first, 0, kloff);
    else
      load_chunk<D, TILES>(ring[0], make_rsrc(Kc, (uint32_t)first * ROW), make_rsrc(Vc, (uint32_t)first * ROW), 0,
                           r16, g4);
  }

  int n = p.len[s];
  n = n < 0 ? 0 : (n > p.cap ? p.cap : n);
  const bool append = kn != nullptr && n >= 1;
  // The new token goes to slot n-1. Its K and V rows are loaded once, as the
  // one-key tile below, and written to the cache from those registers once
  // the unit's other loads are in flight, so no load-to-store round trip
  // precedes them. Reads of the cache stop at slot n-2.
  const bool put_pos = append && p.pos != nullptr && p.new_pos != nullptr;
  const int32_t npos = put_pos ? p.new_pos[s] : 0;
  const int ncache = append ? n - 1 : n;

  // Merge: the partial records of this wave's rows, piece k at stride
  // S*L*Hq records, G contiguous records each. The first merge_pf pieces
  // are copied into LDS now (buffer-to-LDS loads, 1 KiB per instruction) so
  // the epilogue does not wait on them.
  constexpr int RF = kRecFloats<D>;
  int npieces = 0, pf = 0;
  const size_t rstride = (size_t)p.S * p.L * p.Hq * RF;
  const float *rbase = nullptr;
  if constexpr (MERGE) {
    const long ug = ((long)((s / p.C) * p.L + l) * p.Hkv + h) * p.plen;
    npieces = (int)((ug + p.plen - 1) / p.span - ug / p.span) + 1;
    pf = npieces < p.merge_pf ? npieces : p.merge_pf;
    rbase = p.ws + (((size_t)s * p.L + l) * p.Hq + qh0) * RF;
#if defined(__HIP_DEVICE_COMPILE__)
    for (int k = 0; k < pf; k++) {
      const rsrc_t rr = make_rsrc(rbase + k * rstride, (uint32_t)G * RF * 4u);
      for (int j = 0; j < p.merge_blk / 256; j++)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rr, (lds_void_t *)(pbuf + k * p.merge_blk + j * 256), 16,
                                                 (uint32_t)(j * 1024 + lane * 16), 0, 0, 0);
    }
#endif
  }

  // Observation-window step of this sequence?
  const int wstart = p.B + p.buffer + 2 - p.W;
  const bool win = !MERGE && p.scores != nullptr && n >= wstart;
  const int ldx = (p.cap + 63) & ~63;
  float *xs = smem + (KL ? kl_ring<D, TILES, DEPTH> / sizeof(float) : 0);  // [G][ldx] logits of window steps
  float *stat = xs + G * ldx;       // [16] max, [16] 1/sum

  const float sl2 = p.scale * kLog2e;
  RowState st{kNegInf, 0.0f};
  float4_t o[NB];
#pragma unroll
  for (int b = 0; b < NB; b++) o[b] = float4_t{0.f, 0.f, 0.f, 0.f};

  const rsrc_t Kr = make_rsrc(Kc, (uint32_t)ncache * ROW);
  const rsrc_t Vr = make_rsrc(Vc, (uint32_t)ncache * ROW);
  // One chunk: c holds the value rows (and, without KL, the key rows); with
  // KL the key rows are in the LDS slot `kslot`.
  auto process = [&](auto &c, const char *kslot, int c0, int nlim) {
    if (!MERGE && c0 == 0 && nlim < CH) {
      // The first chunk was read before the live length was known.
#pragma unroll
      for (int t = 0; t < TILES; t++)
#pragma unroll
        for (int cc = 0; cc < 4; cc++)
          if (t * 16 + 4 * g4 + cc >= nlim)
#pragma unroll
            for (int w = 0; w < Geo<D>::VW; w++) c.v[t][cc][w] = 0u;
    }
    float x[TILES][4];
    if constexpr (KL)
      chunk_logits_lds<D, TILES>(kslot, qop, x, c0, nlim, r16, g4, sl2, c0 + CH > nlim);
    else
      chunk_logits<D, TILES>(c, qop, x, c0, nlim, g4, sl2, c0 + CH > nlim);
    if (win && r16 < G) {
#pragma unroll
      for (int t = 0; t < TILES; t++)
        *reinterpret_cast<float4_t *>(xs + r16 * ldx + c0 + t * 16 + 4 * g4) =
            float4_t{x[t][0], x[t][1], x[t][2], x[t][3]};
    }
    softmax_pv<D, TILES, true>(x, st, o, c.v, g4);
  };

  // The stored scores of window steps that accumulate are prefetched now,
  // behind the loads issued above; the new token's tile is processed first
  // (key order does not matter to the online softmax).
  constexpr int PRE = 5;  // stored scores prefetched per lane (slots < 320)
  const bool accumulate = win && n != wstart;
  float old[PRE];
  float *sc = win ? p.scores + (size_t)unit * p.cap : nullptr;
  if (accumulate) {
    const rsrc_t Sr = make_rsrc(sc, (uint32_t)(n - 1) * 4u);
#pragma unroll
    for (int k = 0; k < PRE; k++)
      old[k] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(Sr, (uint32_t)(lane + 64 * k) * 4u, 0, 0));
  }
  float xnew = kNegInf;  // the new token's logit, stored after the tail chunk's masked ones
  auto new_token = [&]() {
    if (append) {
      // Cache rows of the new token from the tile's registers: K row 0 is held
      // by the lanes with r16 == 0 (d = 32i + 8 g4), V row 0 by the lanes with
      // g4 == 0 (d = r16 D/16). Every store of this kernel (these rows, the
      // outputs, the score row) carries the non-temporal hint: nothing in the
      // launch reads them back, and streaming them past the caches took 4-6%
      // off the whole launch at the 72B and 7B evicted-cache shapes.
      if (r16 == 0) {
#pragma unroll
        for (int i = 0; i < Geo<D>::NLD; i++)
          __builtin_nontemporal_store(cn.k[0][i],
                                      reinterpret_cast<u32x4 *>(Kc + (size_t)(n - 1) * D + 32 * i + 8 * g4));
      }
      if (g4 == 0) {
        bf16_t *vd = Vc + (size_t)(n - 1) * D + r16 * NB;
        if constexpr (D == 128)
          __builtin_nontemporal_store(u32x4{cn.v[0][0][0], cn.v[0][0][1], cn.v[0][0][2], cn.v[0][0][3]},
                                      reinterpret_cast<u32x4 *>(vd));
        else
          __builtin_nontemporal_store(u32x2{cn.v[0][0][0], cn.v[0][0][1]}, reinterpret_cast<u32x2 *>(vd));
      }
      if (put_pos && lane == 16) __builtin_nontemporal_store(npos, p.pos + (size_t)unit * p.cap + n - 1);
      float x[1][4];
      chunk_logits<D, 1>(cn, qop, x, 0, 1, g4, sl2, true);
      xnew = x[0][0];
      softmax_pv<D, 1, true>(x, st, o, cn.v, g4);
    }
  };
  if constexpr (MERGE) {
    if constexpr (KL)
      load_chunk_lds<D, TILES>(vring[0], kring, Kc, Vc, ncache, 0, kloff);
    else
      load_chunk<D, TILES>(ring[0], Kr, Vr, 0, r16, g4);
  }
  if constexpr (KL)
    stream_chunks_lds<D, TILES, DEPTH>(vring, kring, Kc, Vc, 0, ncache, kloff, new_token,
                                       [&](VChunk<D, TILES> &c, const char *slot, int c0) { process(c, slot, c0, ncache); });
  else
    stream_chunks_from<D, TILES, DEPTH>(ring, Kr, Vr, 0, ncache, r16, g4, new_token,
                                        [&](KVChunk<D, TILES> &c, int c0) { process(c, nullptr, c0, ncache); });
#if defined(__HIP_DEVICE_COMPILE__)
  if constexpr (KL) __builtin_amdgcn_s_waitcnt(0);  // no buffer-to-LDS load outlives the stream
#endif
  if (append && win && r16 < G && g4 == 0) xs[r16 * ldx + n - 1] = xnew;

  float z = st.zl;
  z += shfl_xor(z, 16);
  z += shfl_xor(z, 32);

  bf16_t *out = static_cast<bf16_t *>(p.out);
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const int row = 4 * g4 + i;
    float zi = __shfl(z, row, kWave);
    if constexpr (MERGE) {
      // Log-sum-exp merge with the context partials of this row:
      // record = (max, sum, -, -, o[D] / sum) in the log2 domain.
      const float mi = __shfl(st.m, row, kWave);
      if (i == 0) wait_vm0();  // the LDS copies of the partials have landed
      if (row < G) {
        if (npieces <= kFastPieces && npieces <= pf) {
          // Every piece is in LDS: all of its reads are issued before any is
          // used, so the row's merge costs one LDS round trip.
          float rm[kFastPieces], rs[kFastPieces];
          uint32_t hv[kFastPieces][NB / 2];
#pragma unroll
          for (int k = 0; k < kFastPieces; k++) {
            if (k < npieces) {
              const float *r = pbuf + k * p.merge_blk + row * RF;
              const float2_t ms = *reinterpret_cast<const float2_t *>(r);
              rm[k] = ms.x;
              rs[k] = ms.y;
              if constexpr (D == 128) {
                const u32x4 x = *reinterpret_cast<const u32x4 *>(r + 4 + r16 * (NB / 2));
                hv[k][0] = x.x; hv[k][1] = x.y; hv[k][2] = x.z; hv[k][3] = x.w;
              } else {
                const u32x2 x = *reinterpret_cast<const u32x2 *>(r + 4 + r16 * (NB / 2));
                hv[k][0] = x.x; hv[k][1] = x.y;
              }
            } else {
              rm[k] = kNegInf;
              rs[k] = 0.0f;
#pragma unroll
              for (int b = 0; b < NB / 2; b++) hv[k][b] = 0u;
            }
          }
          float M = mi;
#pragma unroll
          for (int k = 0; k < kFastPieces; k++) M = fmaxf(M, rm[k]);
          const float wown = fast_exp2(mi - M);
          zi *= wown;
#pragma unroll
          for (int b = 0; b < NB; b++) o[b][i] *= wown;
#pragma unroll
          for (int k = 0; k < kFastPieces; k++) {
            const float w = rm[k] == kNegInf ? 0.0f : rs[k] * fast_exp2(rm[k] - M);
            zi += w;
#pragma unroll
            for (int b = 0; b < NB / 2; b++) {
              o[2 * b][i] += f16_lo(hv[k][b]) * w;
              o[2 * b + 1][i] += f16_hi(hv[k][b]) * w;
            }
          }
        } else {
        // Pieces k < pf from LDS, the others from the workspace, in loops of
        // their own so that each reads through its own memory path (one loop
        // over a pointer into either would read through flat addressing and
        // wait for every access in turn).
        float M = mi;
        for (int k = 0; k < pf; k++) M = fmaxf(M, pbuf[k * p.merge_blk + row * RF]);
        for (int k = pf; k < npieces; k++) M = fmaxf(M, rbase[k * rstride + row * RF]);
        const float wown = fast_exp2(mi - M);
        zi *= wown;
#pragma unroll
        for (int b = 0; b < NB; b++) o[b][i] *= wown;
        auto fold = [&](const float *r) {
          const float mk = r[0];
          const float w = mk == kNegInf ? 0.0f : r[1] * fast_exp2(mk - M);
          zi += w;
          // The lane's NB columns: NB float16 at float slot 4 + r16 * NB / 2.
          uint32_t hv[NB / 2];
          if constexpr (D == 128) {
            const u32x4 x = *reinterpret_cast<const u32x4 *>(r + 4 + r16 * (NB / 2));
            hv[0] = x.x; hv[1] = x.y; hv[2] = x.z; hv[3] = x.w;
          } else {
            const u32x2 x = *reinterpret_cast<const u32x2 *>(r + 4 + r16 * (NB / 2));
            hv[0] = x.x; hv[1] = x.y;
          }
#pragma unroll
          for (int b = 0; b < NB / 2; b++) {
            o[2 * b][i] += f16_lo(hv[b]) * w;
            o[2 * b + 1][i] += f16_hi(hv[b]) * w;
          }
        };
        for (int k = 0; k < pf; k++) fold(pbuf + k * p.merge_blk + row * RF);
        for (int k = pf; k < npieces; k++) fold(rbase + k * rstride + row * RF);
        }
      }
    }
    if (row < G) {
      const float inv = 1.0f / zi;
      uint32_t w[NB / 2];
#pragma unroll
      for (int b = 0; b < NB / 2; b++) w[b] = pack_bf16x2(o[2 * b][i] * inv, o[2 * b + 1][i] * inv);
      bf16_t *dst = out + (qrow0 + row) * D + r16 * NB;
      if constexpr (D == 128)
        __builtin_nontemporal_store(u32x4{w[0], w[1], w[2], w[3]}, reinterpret_cast<u32x4 *>(dst));
      else
        __builtin_nontemporal_store(u32x2{w[0], w[1]}, reinterpret_cast<u32x2 *>(dst));
    }
  }
  if constexpr (!MERGE) {
    if (win) {
      if (g4 == 0 && r16 < G) {
        stat[r16] = st.m;
        stat[16 + r16] = 1.0f / z;
      }
      __syncthreads();
      // Slot n-1 (the new token) and the first window step store; older slots
      // add to the stored score (prefetched above for the first PRE*64 slots).
#pragma unroll
      for (int k = 0; k < PRE; k++) {
        const int j = lane + 64 * k;
        if (j < n) {
          float r = 0.0f;
          for (int g = 0; g < G; g++) r += fast_exp2(xs[g * ldx + j] - stat[g]) * stat[16 + g];
          __builtin_nontemporal_store((accumulate && j < n - 1) ? old[k] + r : r, sc + j);
        }
      }
      for (int j = lane + 64 * PRE; j < n; j += kWave) {
        float r = 0.0f;
        for (int g = 0; g < G; g++) r += fast_exp2(xs[g * ldx + j] - stat[g]) * stat[16 + g];
        __builtin_nontemporal_store((accumulate && j < n - 1) ? sc[j] + r : r, sc + j);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Prefix kernel: each wave walks its span of the flattened (prefix, layer,
// KV head, key) space one unit segment at a time; RB row blocks of 16 rows
// hold the C*G query rows (candidate c, head g) sharing the prefix, so each
// prefix byte is read once per step for all of them. Same double-buffered
// chunk stream as the own-cache kernel. `wave` is the wave's index in the
// plan (its span is keys [wave * span, (wave + 1) * span)).
//
// deferred: records of the wave's first segment when more follow,
// [rows][4 + D/2] floats in LDS, written to the workspace once the span is
// done. Stores to HBM in the middle of a wave's read stream cost far more
// than their bytes (measured: about 6% of the kernel's time), so every record
// store waits for the end of the wave.
template <int D, int RB, int TILES, int DEPTH>
__device__ __forceinline__ void prefix_wave(const AttnParams &p, const int wave, float *deferred) {
  constexpr int CH = 16 * TILES;
  constexpr int NB = Geo<D>::NB;
  constexpr uint32_t ROW = D * 2;
  const long total = (long)p.P * p.L * p.Hkv * p.plen;
  const long g0 = (long)wave * p.span;
  const long g1 = g0 + p.span < total ? g0 + p.span : total;
  const int lane = threadIdx.x;
  const int r16 = lane & 15;
  const int g4 = lane >> 4;
  const int G = p.G;
  const int rows = p.C * G;
  int dunit = -1, dsplit = 0;

  // This wave's keys [g0, g1) of the flattened (unit, key) space, one segment
  // per unit it touches; each segment leaves one partial record per row.
#pragma clang loop unroll(disable)
  for (long g = g0; g < g1;) {
  const int unit = (int)(g / p.plen);  // ((pp * L) + l) * Hkv + h
  const int k0 = (int)(g - (long)unit * p.plen);
  const int k1 = (int)((long)p.plen < k0 + (g1 - g) ? (long)p.plen : k0 + (g1 - g));
  const int split = wave - (int)((long)unit * p.plen / p.span);  // piece index within the unit
  g += k1 - k0;
  const int h = unit % p.Hkv;
  const int pl = unit / p.Hkv;
  const int l = pl % p.L;
  const int pp = pl / p.L;

  const bf16_t *Kp = static_cast<const bf16_t *>(p.pk) + (size_t)unit * p.plen * D;
  const bf16_t *Vp = static_cast<const bf16_t *>(p.pv) + (size_t)unit * p.plen * D;

  short4_t qop[RB][NB];
#pragma unroll
  for (int rb = 0; rb < RB; rb++) {
    const int rho = rb * 16 + r16;
    const bf16_t *qrow = nullptr;
    if (rho < rows) {
      const int c = rho / G, g = rho % G;
      const int s = pp * p.C + c;
      qrow = static_cast<const bf16_t *>(p.q) + (((size_t)s * p.L + l) * p.Hq + h * G + g) * D;
    }
    load_qop<D>(qrow, g4, qop[rb]);
  }

  const float sl2 = p.scale * kLog2e;
  RowState st[RB];
  float4_t o[RB][NB];
#pragma unroll
  for (int rb = 0; rb < RB; rb++) {
    st[rb] = RowState{kNegInf, 0.0f};
#pragma unroll
    for (int b = 0; b < NB; b++) o[rb][b] = float4_t{0.f, 0.f, 0.f, 0.f};
  }

  // Byte range covers keys [0, k1); chunk offsets are absolute key indices.
  const rsrc_t Kr = make_rsrc(Kp, (uint32_t)(k1 > 0 ? k1 : 0) * ROW);
  const rsrc_t Vr = make_rsrc(Vp, (uint32_t)(k1 > 0 ? k1 : 0) * ROW);
  auto process = [&](const KVChunk<D, TILES> &c, int c0) {
    const bool tail = c0 + CH > k1;
    if constexpr (RB == 2 || RB == 3) {
      short4_t vo[TILES][NB];
      make_vops<D, TILES>(c.v, vo);
#pragma unroll
      for (int rb = 0; rb < RB; rb++) {
        float x[TILES][4];
        chunk_logits<D, TILES>(c, qop[rb], x, c0, k1, g4, sl2, tail);
        softmax_pv<D, TILES, true>(x, st[rb], o[rb], vo, g4);
      }
    } else {
#pragma unroll
      for (int rb = 0; rb < RB; rb++) {
        float x[TILES][4];
        chunk_logits<D, TILES>(c, qop[rb], x, c0, k1, g4, sl2, tail);
        softmax_pv<D, TILES, true>(x, st[rb], o[rb], c.v, g4);
      }
    }
  };
  stream_chunks<D, TILES, DEPTH>(Kr, Vr, k0, k1, r16, g4, [] {}, process);

  // The segment's records: to LDS if it is the first of several, else to
  // the workspace.
  const bool defer = dunit < 0 && g < g1;
  if (defer) {
    dunit = unit;
    dsplit = split;
  }
#pragma unroll
  for (int rb = 0; rb < RB; rb++) {
    float z = st[rb].zl;
    z += shfl_xor(z, 16);
    z += shfl_xor(z, 32);
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const int rl = 4 * g4 + i;
      const float mi = __shfl(st[rb].m, rl, kWave);
      const float zi = __shfl(z, rl, kWave);
      const int rho = rb * 16 + rl;
      if (rho < rows) {
        // One store of the lane's NB consecutive columns of o / sum as
        // float16 (16 bytes at D = 128; records are 16-byte multiples), and
        // (max, sum) from the first lane of the row.
        const float inv = zi > 0.f ? 1.0f / zi : 0.f;
        auto put = [&](float *r) {
          if (r16 == 0) *reinterpret_cast<float2_t *>(r) = float2_t{mi, zi};
          uint32_t hv[NB / 2];
#pragma unroll
          for (int b = 0; b < NB / 2; b++) hv[b] = pack_f16x2(o[rb][2 * b][i] * inv, o[rb][2 * b + 1][i] * inv);
          if constexpr (D == 128)
            *reinterpret_cast<u32x4 *>(r + 4 + r16 * (NB / 2)) = u32x4{hv[0], hv[1], hv[2], hv[3]};
          else
            *reinterpret_cast<u32x2 *>(r + 4 + r16 * (NB / 2)) = u32x2{hv[0], hv[1]};
        };
        if (defer) {
          put(deferred + (size_t)rho * kRecFloats<D>);
        } else {
          const int c = rho / G, g = rho % G;
          const int s = pp * p.C + c;
          put(p.ws + ((((size_t)split * p.S + s) * p.L + l) * p.Hq + h * G + g) * kRecFloats<D>);
        }
      }
    }
  }
  }  // segments

  // Write out the deferred records: the G records of a candidate are
  // contiguous in the workspace (record ((split * S + s) * L + l) * Hq + h G + g).
  if (dunit >= 0) {
    __syncthreads();
    const int h = dunit % p.Hkv;
    const int pl = dunit / p.Hkv;
    const int l = pl % p.L;
    const int pp = pl / p.L;
    const int per_c = G * kRecFloats<D> / 4;  // 16-byte vectors per candidate
    const float4_t *src = reinterpret_cast<const float4_t *>(deferred);
    for (int u = lane; u < p.C * per_c; u += kWave) {
      const int c = u / per_c;
      const size_t rec0 = (((size_t)dsplit * p.S + pp * p.C + c) * p.L + l) * p.Hq + h * G;
      reinterpret_cast<float4_t *>(p.ws + rec0 * kRecFloats<D>)[u - c * per_c] = src[u];
    }
  }
}

template <int D, int RB, int TILES, int DEPTH>
__global__ __launch_bounds__(64) void attn_prefix_bf16(AttnParams p) {
  extern __shared__ float deferred[];
  prefix_wave<D, RB, TILES, DEPTH>(p, blockIdx.x, deferred);
}

// One logit row of the batch (global row g) by one wave, the variant picked at
// run time from the batch's logit type and sampler; cand: kSampleRowLds bytes
// of LDS owned by the wave.
__device__ __forceinline__ void entropy_row_any(const EntropyBatch &e, int g, int lane, uint64_t *cand) {
  const int k = batch_set(e, g);
  const EntropyParams &s = e.set[k];
  const int row = g - e.row0[k];
  if (s.top_k > 0) {
    if (s.dtype == 0) entropy_sample_row_wave<float, 4>(s, row, lane, cand);
    else entropy_sample_row_wave<bf16_t, 8>(s, row, lane, cand);
  } else {
    if (s.dtype == 0) entropy_row_wave<float, 6>(s, row, lane);
    else entropy_row_wave<bf16_t, 12>(s, row, lane);
  }
}

// The prefix kernel with the step's logit rows in front: the first
// e.row0[e.nsets] workgroups are one wave per row (entropy, detector update
// and, with a sampler, the token draw), dispatched first so that they stream
// their rows beside the context waves; the plan then has that many fewer
// context waves, so that both fit on the chip in one round.
template <int D, int RB, int TILES, int DEPTH>
__global__ __launch_bounds__(64) void attn_prefix_rows_bf16(AttnParams p, EntropyBatch e) {
  extern __shared__ float deferred[];
  const int rows = e.row0[e.nsets];
  if ((int)blockIdx.x < rows) {
    entropy_row_any(e, blockIdx.x, threadIdx.x, reinterpret_cast<uint64_t *>(deferred));
    return;
  }
  prefix_wave<D, RB, TILES, DEPTH>(p, blockIdx.x - rows, deferred);
}

#if !KVR_ATTN_WIDE
// ---------------------------------------------------------------------------
// float32 path: one wave per (sequence, layer, KV head), VALU arithmetic.
// LDS: q rows [G][D], logits [G][nt_max], stats [2][16].
__global__ __launch_bounds__(64) void attn_f32(AttnParams p, int nt_max) {
  extern __shared__ float smem[];
  const int unit = blockIdx.x;
  const int h = unit % p.Hkv;
  const int sl = unit / p.Hkv;
  const int l = sl % p.L;
  const int s = sl / p.L;
  const int lane = threadIdx.x;
  const int G = p.G, D = p.D;
  int n = p.len[s];
  n = n < 0 ? 0 : (n > p.cap ? p.cap : n);
  const int npre = p.P > 0 ? p.plen : 0;
  const int nt = npre + n;
  const size_t ubase = (size_t)unit * p.cap * D;
  float *Kc = static_cast<float *>(p.k) + ubase;
  float *Vc = static_cast<float *>(p.v) + ubase;
  const float *kn = p.k_new ? static_cast<const float *>(p.k_new) + (size_t)unit * D : nullptr;
  const float *vn = p.v_new ? static_cast<const float *>(p.v_new) + (size_t)unit * D : nullptr;
  const float *Kp = nullptr, *Vp = nullptr;
  if (p.P > 0) {
    const int pp = s / p.C;
    const size_t pbase = (((size_t)pp * p.L + l) * p.Hkv + h) * (size_t)p.plen * D;
    Kp = static_cast<const float *>(p.pk) + pbase;
    Vp = static_cast<const float *>(p.pv) + pbase;
  }
  if (kn && n >= 1) {
    for (int d = lane; d < D; d += kWave) {
      Kc[(size_t)(n - 1) * D + d] = kn[d];
      Vc[(size_t)(n - 1) * D + d] = vn[d];
    }
    if (lane == 0 && p.pos && p.new_pos) p.pos[(size_t)unit * p.cap + n - 1] = p.new_pos[s];
  }
  auto krow = [&](int j) -> const float * {
    if (j < npre) return Kp + (size_t)j * D;
    const int js = j - npre;
    return (kn && js == n - 1) ? kn : Kc + (size_t)js * D;
  };
  auto vrow = [&](int j) -> const float * {
    if (j < npre) return Vp + (size_t)j * D;
    const int js = j - npre;
    return (vn && js == n - 1) ? vn : Vc + (size_t)js * D;
  };
  float *qs = smem;
  float *xs = smem + G * D;
  float *stat = xs + (size_t)G * nt_max;
  const size_t qrow0 = ((size_t)s * p.L + l) * p.Hq + h * G;
  for (int e = lane; e < G * D; e += kWave) qs[e] = static_cast<const float *>(p.q)[qrow0 * D + e];
  __syncthreads();
  for (int g = 0; g < G; g++) {
    float mloc = kNegInf;
    for (int j = lane; j < nt; j += kWave) {
      const float *kr = krow(j);
      float dot = 0.f;
      for (int d = 0; d < D; d++) dot = fmaf(qs[g * D + d], kr[d], dot);
      const float x = dot * p.scale;
      xs[g * nt_max + j] = x;
      mloc = fmaxf(mloc, x);
    }
    const float m = wave_max(mloc);
    float zloc = 0.f;
    for (int j = lane; j < nt; j += kWave) zloc += expf(xs[g * nt_max + j] - m);
    const float z = wave_sum(zloc);
    if (lane == 0) { stat[g] = m; stat[16 + g] = 1.0f / z; }
  }
  __syncthreads();
  float *out = static_cast<float *>(p.out);
  for (int g = 0; g < G; g++) {
    const float m = stat[g], iz = stat[16 + g];
    for (int d = lane; d < D; d += kWave) {
      float acc = 0.f;
      for (int j = 0; j < nt; j++) acc = fmaf(expf(xs[g * nt_max + j] - m) * iz, vrow(j)[d], acc);
      out[(qrow0 + g) * D + d] = acc;
    }
  }
  const int wstart = p.B + p.buffer + 2 - p.W;
  if (p.scores != nullptr && p.P == 0 && n >= wstart) {
    const bool first = n == wstart;
    float *sc = p.scores + (size_t)unit * p.cap;
    for (int j = lane; j < n; j += kWave) {
      float r = 0.f;
      for (int g = 0; g < G; g++) r += expf(xs[g * nt_max + j] - stat[g]) * stat[16 + g];
      if (first || j == n - 1)
        sc[j] = r;
      else
        sc[j] += r;
    }
  }
}
#endif  // !KVR_ATTN_WIDE

// LDS of a context-kernel wave: the deferred records of RB * 16 rows. A
// logit-row wave of the same launch uses the first kSampleRowLds bytes of it.
template <int D>
size_t prefix_lds_bytes(int rb) {
  return (size_t)rb * 16 * kRecFloats<D> * sizeof(float);
}
static_assert(16 * kRecFloats<64> * sizeof(float) >= kSampleRowLds, "row waves fit the context kernel's LDS");

// The context kernel, with the entropy rows of `e` (nullptr: none) in front.
template <int D, int RB, int TILES>
void launch_prefix(const AttnParams &p, const EntropyBatch *e, hipStream_t stream) {
  const size_t lds = prefix_lds_bytes<D>(RB);
  if (e)
    hipLaunchKernelGGL((attn_prefix_rows_bf16<D, RB, TILES, 2>), dim3(e->row0[e->nsets] + p.nwaves), dim3(64), lds,
                       stream, p, *e);
  else
    hipLaunchKernelGGL((attn_prefix_bf16<D, RB, TILES, 2>), dim3(p.nwaves), dim3(64), lds, stream, p);
}

// The evicted-cache kernel with the entropy rows of `e` (nullptr: none) in
// front of its units.
template <int D, int TILES, int DEPTH, bool KL>
void launch_own(const AttnParams &p, const EntropyBatch *e, size_t lds, hipStream_t stream) {
  const int rows = e ? e->row0[e->nsets] : 0;
  const dim3 grid(rows + p.S * p.L * p.Hkv);
  const EntropyBatch none{};
  const bool f32 = e && e->set[0].dtype == 0;
  const bool sample = e && e->set[0].top_k > 0;
  if (sample && lds < kSampleRowLds) lds = kSampleRowLds;  // the row waves' candidate buffers
  if (!e)
    hipLaunchKernelGGL((attn_cache_bf16<D, false, TILES, DEPTH, KL, 0>), grid, dim3(64), lds, stream, p, none);
  else if (sample && f32)
    hipLaunchKernelGGL((attn_cache_bf16<D, false, TILES, DEPTH, KL, 4>), grid, dim3(64), lds, stream, p, *e);
  else if (sample)
    hipLaunchKernelGGL((attn_cache_bf16<D, false, TILES, DEPTH, KL, 3>), grid, dim3(64), lds, stream, p, *e);
  else if (f32)
    hipLaunchKernelGGL((attn_cache_bf16<D, false, TILES, DEPTH, KL, 2>), grid, dim3(64), lds, stream, p, *e);
  else
    hipLaunchKernelGGL((attn_cache_bf16<D, false, TILES, DEPTH, KL, 1>), grid, dim3(64), lds, stream, p, *e);
}

template <int D>
hipError_t launch_bf16(const AttnParams &p_in, const EntropyBatch *ent, hipStream_t stream) {
  AttnParams p = p_in;
  if (p.P > 0) {
    // LDS for the suffix kernel's prefetched partials: whole 1 KiB blocks per
    // piece, at most 16 KiB per wave (8 waves per CU then use 128 of 160 KiB).
    p.merge_blk = (p.G * kRecFloats<D> * 4 + 1023) / 1024 * 256;
    const int fit = (int)(kMergePrefetchBytes / (p.merge_blk * 4));
    p.merge_pf = p.nsplit < fit ? p.nsplit : fit;
  }
  const dim3 units(p.S * p.L * p.Hkv);
  if (p.P == 0) {
    // Register-resident keys (the fallback when the LDS ring and the window
    // logits do not fit): at D = 128 the kernel asks for at least 26 KiB of
    // LDS, which caps it at 6 single-wave workgroups per CU (160 KiB) instead
    // of the 8 its registers allow: fewer concurrent short K/V streams
    // measured 2.5-3.5% faster (5 per CU lost at short caches, 7 matched 6).
    const size_t logits = p.scores ? ((size_t)p.G * ((p.cap + 63) & ~63) + 32) * sizeof(float) : 0;
    const size_t lds_min = D == 128 ? kBaseLdsFloor : 0;
    constexpr size_t ring = kl_ring<D, kKlTiles, kKlDepth>;
    if (ring + logits <= kMaxLds) {
      // Key rows through the LDS ring. No floor here: with the keys in LDS,
      // 7-8 workgroups per CU (registers: 172) measured 1-1.5% faster than the
      // 6 of a 26 KiB floor on the 7B shapes and equal on the 72B shape.
      launch_own<D, kKlTiles, kKlDepth, true>(p, ent, ring + logits, stream);
    } else {
      launch_own<D, 2, 2, false>(p, ent, logits > lds_min ? logits : lds_min, stream);
    }
    return hipGetLastError();
  }
  // Context splits first (with the logit rows, if any); the suffix kernel
  // then merges their partials.
  switch ((p.C * p.G + 15) / 16) {
    case 1: launch_prefix<D, 1, 2>(p, ent, stream); break;
    case 2: launch_prefix<D, 2, 2>(p, ent, stream); break;
    case 3: launch_prefix_wide(D, 3, p, ent, stream); break;
    case 4: launch_prefix_wide(D, 4, p, ent, stream); break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t pre = (size_t)p.merge_pf * p.merge_blk * sizeof(float);
  constexpr size_t ring = kl_ring<D, kKlTiles, kKlDepth>;
  if constexpr (kSuffixKl)
    hipLaunchKernelGGL((attn_cache_bf16<D, true, kKlTiles, kKlDepth, true>), units, dim3(64), ring + pre, stream, p,
                       EntropyBatch{});
  else
    hipLaunchKernelGGL((attn_cache_bf16<D, true, 2, 2>), units, dim3(64), pre, stream, p, EntropyBatch{});
  return hipGetLastError();
}

// Whole logit rows, one wave per row, as a kernel of its own (the entropy
// rows of a float32-cache launch, whose attention kernel has no such lanes).
template <typename T, bool SAMPLE>
__global__ __launch_bounds__(64) void entropy_rows_kernel(EntropyBatch e) {
  extern __shared__ uint64_t cand[];
  const int g = blockIdx.x;
  const int k = batch_set(e, g);
  if constexpr (SAMPLE)
    entropy_sample_row_wave<T, sizeof(T) == 2 ? 8 : 4>(e.set[k], g - e.row0[k], threadIdx.x, cand);
  else
    entropy_row_wave<T, sizeof(T) == 2 ? 12 : 6>(e.set[k], g - e.row0[k], threadIdx.x);
}

}  // namespace

#if !KVR_ATTN_WIDE
size_t f32_attn_lds_bytes(int G, int D, int plen, int cap) {
  return ((size_t)G * D + (size_t)G * (plen + cap) + 32) * sizeof(float);
}
#endif

namespace {

// Waves of one prefix-kernel instantiation (ROWS: the one with logit rows in
// front) that fit on the device at once (occupancy per CU x CU count), looked
// up once per instantiation.
template <int D, int RB, int TILES, bool ROWS>
int prefix_slots() {
  static std::atomic<int> cached{0};
  int v = cached.load(std::memory_order_relaxed);
  if (v > 0) return v;
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  hipError_t e;
  if constexpr (ROWS)
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, attn_prefix_rows_bf16<D, RB, TILES, 2>, 64,
                                                     prefix_lds_bytes<D>(RB));
  else
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, attn_prefix_bf16<D, RB, TILES, 2>, 64,
                                                     prefix_lds_bytes<D>(RB));
  if (e != hipSuccess || per_cu <= 0) per_cu = 4;
  v = cus * per_cu;
  cached.store(v, std::memory_order_relaxed);
  return v;
}

#if !KVR_ATTN_WIDE
template <int D, bool ROWS>
int prefix_slots_for(int rb) {
  switch (rb) {
    case 1: return prefix_slots<D, 1, 2, ROWS>();
    case 2: return prefix_slots<D, 2, 2, ROWS>();
    default: return (int)prefix_slots_wide(D, rb, ROWS);
  }
}

long slots_for(int D, int rb, bool rows) {
  if (D == 128) return rows ? prefix_slots_for<128, true>(rb) : prefix_slots_for<128, false>(rb);
  return rows ? prefix_slots_for<64, true>(rb) : prefix_slots_for<64, false>(rb);
}
#endif  // !KVR_ATTN_WIDE

}  // namespace

#if !KVR_ATTN_WIDE

void plan_prefix_splits(int D, int P, int L, int Hkv, int plen, int rows, int ent_rows, int *nsplit, int *span,
                        int *nwaves) {
  // One round of waves: as many as fit on the chip at once, each taking an
  // equal span (whole 32-key chunks, at least 512 keys) of the flattened
  // (prefix, layer, KV head, key) space. A unit of plen keys is then covered
  // by at most ceil(plen / span) + 1 spans. Logit-row waves in the same
  // launch take their slots first (the context waves keep at least half), and
  // the context waves never outnumber those of the plan without rows, so that
  // plan's workspace size covers both.
  const int rb = (rows + 15) / 16;
  const long total = (long)P * L * Hkv * plen;
  long slots = slots_for(D, rb, false);
  if (ent_rows > 0) {
    const long with_rows = slots_for(D, rb, true);
    const long all = with_rows < slots ? with_rows : slots;
    slots = all - ent_rows > all / 2 ? all - ent_rows : all / 2;
    if (slots < 1) slots = 1;
  }
  long sp = (total + slots - 1) / slots;
  sp = (sp + 31) / 32 * 32;
  if (sp < 512) sp = 512;
  const long nw = (total + sp - 1) / sp;
  *span = (int)sp;
  *nwaves = (int)nw;
  *nsplit = (int)((plen + sp - 1) / sp + 1);
}

size_t attn_workspace_bytes(int S, int L, int Hq, int D, int nsplit) {
  return (size_t)nsplit * S * L * Hq * (D == 128 ? kRecFloats<128> : kRecFloats<64>) * sizeof(float);
}

hipError_t launch_decode_attn(const AttnParams &p, const EntropyBatch *ent, hipStream_t stream) {
  if (p.dtype == 0) {
    const int nt_max = (p.P > 0 ? p.plen : 0) + p.cap;
    const size_t lds = f32_attn_lds_bytes(p.G, p.D, p.P > 0 ? p.plen : 0, p.cap);
    hipLaunchKernelGGL(attn_f32, dim3(p.S * p.L * p.Hkv), dim3(64), lds, stream, p, nt_max);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !ent) return e;
    const dim3 rows(ent->row0[ent->nsets]);
    const bool sample = ent->set[0].top_k > 0;
    const size_t rlds = sample ? kSampleRowLds : 0;
    if (ent->set[0].dtype == 0) {
      if (sample) hipLaunchKernelGGL((entropy_rows_kernel<float, true>), rows, dim3(64), rlds, stream, *ent);
      else hipLaunchKernelGGL((entropy_rows_kernel<float, false>), rows, dim3(64), 0, stream, *ent);
    } else {
      if (sample) hipLaunchKernelGGL((entropy_rows_kernel<bf16_t, true>), rows, dim3(64), rlds, stream, *ent);
      else hipLaunchKernelGGL((entropy_rows_kernel<bf16_t, false>), rows, dim3(64), 0, stream, *ent);
    }
    return hipGetLastError();
  }
  return p.D == 128 ? launch_bf16<128>(p, ent, stream) : launch_bf16<64>(p, ent, stream);
}

#else  // KVR_ATTN_WIDE

void launch_prefix_wide(int D, int rb, const AttnParams &p, const EntropyBatch *e, hipStream_t stream) {
  if (D == 128) {
    if (rb == 3) launch_prefix<128, 3, 1>(p, e, stream);
    else launch_prefix<128, 4, 1>(p, e, stream);
  } else {
    if (rb == 3) launch_prefix<64, 3, 1>(p, e, stream);
    else launch_prefix<64, 4, 1>(p, e, stream);
  }
}

long prefix_slots_wide(int D, int rb, bool rows) {
  if (D == 128) {
    if (rb == 3) return rows ? prefix_slots<128, 3, 1, true>() : prefix_slots<128, 3, 1, false>();
    return rows ? prefix_slots<128, 4, 1, true>() : prefix_slots<128, 4, 1, false>();
  }
  if (rb == 3) return rows ? prefix_slots<64, 3, 1, true>() : prefix_slots<64, 3, 1, false>();
  return rows ? prefix_slots<64, 4, 1, true>() : prefix_slots<64, 4, 1, false>();
}

#endif  // KVR_ATTN_WIDE

}  // namespace kvr
