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
//
// Fused sampler (temperature, top-k, top-p; Sec. 4.1 decoding setup) in the
// same pass. Each wave keeps its best candidates in LDS as 64-bit keys (an
// order-preserving map of the raw logit's bits above the complemented token
// id, so a larger key is a larger logit and, among equal logits, a lower id).
// A candidate must beat the wave's threshold, the k-th best key at its last
// compaction (seeded, in the first round, with the k-th largest of the lanes'
// maxima, which bounds the wave's k-th best logit from below); a batch of 8
// logits per lane in which no lane reaches it costs a few compares and one
// vote. When the buffer would overflow, the wave keeps at most 128 of its best
// and raises the threshold. Thresholds are found bit by bit from the top with
// ballot counts only (compare, ballot, popcount; no cross-lane data movement),
// stopping as soon as the kept count fits. Each split ends
// with its k best keys in the workspace; the per-row merge takes the k best
// of all splits, forms the temperature softmax over them, cuts the nucleus at
// top_p and draws with a Philox4x64-10 uniform (counter (step, row, 0, 0),
// key (seed, 0), top 24 bits of the first word).
#include <hip/hip_runtime.h>

#include <atomic>

#include "entropy_common.h"
#include "sampler_common.h"
#include "kvr_device.h"
#include "kvr_internal.h"

namespace kvr {

// Split partials of the allocation-free entropy entry point: one file-scope
// device array per GPU, held until the process ends. Host code never uses
// its name as an address; it uses the per-device pointer from
// entropy_scratch() below.
__device__ __align__(256) unsigned char scratch[kEntropyScratchBytes];

namespace {

constexpr int kThreads = 256;
constexpr int kU = 10;                      // 8-logit vectors per thread per round (entropy alone)
constexpr int kRoundVecs = kU * kThreads;   // vectors per workgroup per round
// Whole-row workgroups: when a call has at least one row per CU and long
// rows, each row gets one workgroup of kRowThreads threads that reduces it
// completely (entropy and detector in the same kernel, no split partials
// and no merge launch).
constexpr int kRowThreads = 1024;
constexpr int kRowMinRows = 256;
constexpr int kRowMinVecs = 8 * kRowThreads;

// The k best keys of the waves' candidate lists (wave w holds off[w+1]-off[w]
// keys at cand[w * kCandCap ..]) stored unordered to out; returns how many.
template <int NPL, int NW>
__device__ __forceinline__ int gather_select(const uint64_t *cand, const int (&off)[NW + 1], int k, int lane,
                                             uint64_t *out) {
  uint64_t v[NPL];
#pragma unroll
  for (int i = 0; i < NPL; i++) {
    const int j = lane + i * kWave;  // entry j of the concatenated lists
    int w = 0;
#pragma unroll
    for (int q = 1; q < NW; q++) w += j >= off[q];
    v[i] = j < off[NW] ? cand[w * kCandCap + (j - off[w])] : 0;
  }
  const uint64_t thr = select_threshold<NPL>(v, k, k);
  return wave_store_ge<NPL>(out, v, thr, lane);
}

// One workgroup of NT threads per (split, global row of the batch).
// VEC = true: 16-byte loads of 8 elements (row starts 16-byte aligned).
// SAMPLE = true: also collect the split's top_k candidates (always writes
// the split's partials, even unsplit rows, for the sampling merge).
template <typename T, bool VEC, bool SAMPLE, int NT = kThreads>
__global__ __launch_bounds__(NT) void entropy_kernel(EntropyBatch b) {
  __shared__ Tri part[NT / kWave];
  __shared__ uint64_t cand[SAMPLE ? (NT / kWave) * kCandCap : 1];
  __shared__ int cand_n[NT / kWave];
  const int bset = batch_set(b, blockIdx.y);
  const EntropyParams &p = b.set[bset];
  const int row = blockIdx.y - b.row0[bset];
  const int split = blockIdx.x;
  const int splits = gridDim.x;
  const int tid = threadIdx.x;
  const int lane = tid % kWave;
  const int wave = tid / kWave;
  const T *x = static_cast<const T *>(p.logits) + (size_t)row * p.ld;
  const float c = p.inv_temp * kLog2e;
  Cands cs{cand + (SAMPLE ? wave * kCandCap : 0), 0, 1, kNegInf};

  Tri t{kNegInf, 0.f, 0.f};
  if constexpr (VEC) {
    // U vectors of 8 logits per thread per round, all loads issued first and
    // each vector folded as soon as it has arrived, so the arithmetic of the
    // round overlaps its later loads. Entropy alone: 10, so that a split of
    // the 7B / 1.5B vocabularies over 8 workgroups per row is one round. With
    // the sampler: 8, whose lower register count keeps 4 waves per SIMD.
    // Whole-row workgroups keep 10 (20, one round over a 152k bf16 row,
    // measured 3% slower).
    constexpr int U = SAMPLE ? 8 : kU;
    const int nvec = p.V / 8;
    const int per = (nvec + splits - 1) / splits;
    const int v0 = split * per;
    const int v1 = min(v0 + per, nvec);
    // The resource ends where this split's vectors end, so the lanes of a
    // partly used round load nothing instead of fetching the next split.
    const rsrc_t rr = row_rsrc(x, (uint32_t)v1 * 8u * (uint32_t)sizeof(T));
    // The loop bound is the same for every thread (lanes past the end load
    // zeros and skip them), so waves offer sampler candidates in lockstep.
    for (int b0 = v0; b0 < v1; b0 += U * NT) {
      const int base = b0 + tid;
      const bool full = b0 + U * NT <= v1;
      // The loads are issued in vector order (the scheduling barriers keep
      // the compiler from reordering them), so that each fold below waits
      // only for its own vector; the asm statement keeps a load whose value
      // is used under a branch from sinking into it.
      Vec8<T> w[U];
#pragma unroll
      for (int u = 0; u < U; u++) {
        w[u].load(rr, base + u * NT);
        __builtin_amdgcn_sched_barrier(0);
      }
      asm volatile("" ::: "memory");
      if constexpr (SAMPLE) {
        if (b0 == v0) {
          // First round: seed the thresholds from the lanes' maxima.
          float mx = kNegInf;
#pragma unroll
          for (int u = 0; u < U; u++) {
            float a[8];
            w[u].get(a);
            if (base + u * NT < v1)
#pragma unroll
              for (int e = 0; e < 8; e++) mx = vmax(mx, a[e]);
          }
          cand_seed(cs, mx, p.top_k);
        }
      }
#pragma unroll
      for (int u = 0; u < U; u++) {
        float a[8];
        w[u].get(a);
        const int v = base + u * NT;
        const bool ok = full || v < v1;
        if constexpr (SAMPLE) cand_offer(cs, p.top_k, lane, a, (uint32_t)v * 8u, ok ? 8 : 0);
        if (ok) tri_fold8(t, a, c);
      }
    }
    if (split == splits - 1) {
      // The V % 8 trailing logits (one per thread of the first wave).
      const int e = nvec * 8 + tid;
      float a[8] = {kNegInf, kNegInf, kNegInf, kNegInf, kNegInf, kNegInf, kNegInf, kNegInf};
      const bool has = e < p.V;
      if (has) a[0] = load1(x + e);
      if constexpr (SAMPLE) {
        if (wave == 0) cand_offer(cs, p.top_k, lane, a, (uint32_t)e, has ? 1 : 0);
      }
      if (has) {
        float b[1] = {a[0] * c};
        tri_add<1>(t, b);
      }
    }
  } else {
    const int per = (p.V + splits - 1) / splits;
    const int e0 = split * per;
    const int e1 = min(e0 + per, p.V);
    // Every thread runs the same number of iterations so that whole waves
    // offer candidates together.
    for (int eb = e0; eb < e1; eb += NT) {
      const int e = eb + tid;
      const bool has = e < e1;
      float a[8] = {kNegInf, kNegInf, kNegInf, kNegInf, kNegInf, kNegInf, kNegInf, kNegInf};
      if (has) a[0] = load1(x + e);
      if constexpr (SAMPLE) cand_offer(cs, p.top_k, lane, a, (uint32_t)e, has ? 1 : 0);
      if (has) {
        float b[1] = {a[0] * c};
        tri_add<1>(t, b);
      }
    }
  }

#pragma unroll
  for (int msk = 32; msk >= 1; msk >>= 1) {
    Tri o{shfl_xor(t.m, msk), shfl_xor(t.z, msk), shfl_xor(t.s, msk)};
    t = tri_merge(t, o);
  }
  if (lane == 0) part[wave] = t;
  if constexpr (SAMPLE) {
    if (cs.cnt > p.top_k) cand_reduce_any(cs, p.top_k, p.top_k, lane);  // exactly the k best
    if (lane == 0) cand_n[wave] = cs.cnt;
  }
  __syncthreads();
  if constexpr (SAMPLE) {
    // First wave: the k best of the waves' lists go to the workspace.
    if (wave != 0) return;
    constexpr int NW = NT / kWave;
    int off[NW + 1];
    off[0] = 0;
#pragma unroll
    for (int w = 0; w < NW; w++) off[w + 1] = off[w] + cand_n[w];
    uint64_t *keys = reinterpret_cast<uint64_t *>(static_cast<float *>(p.ws) + (size_t)p.R * splits * 4) +
                     ((size_t)row * splits + split) * p.top_k;
    int nw;
    if (off[NW] <= kWave) nw = gather_select<1, NW>(cand, off, p.top_k, lane, keys);
    else if (off[NW] <= 2 * kWave) nw = gather_select<2, NW>(cand, off, p.top_k, lane, keys);
    else nw = gather_select<NW * kTopKMax / kWave, NW>(cand, off, p.top_k, lane, keys);
    for (int q = nw + lane; q < p.top_k; q += kWave) keys[q] = 0;
    if (lane == 0) {
      Tri r = part[0];
#pragma unroll
      for (int w = 1; w < NW; w++) r = tri_merge(r, part[w]);
      reinterpret_cast<float4 *>(p.ws)[(size_t)row * splits + split] = make_float4(r.m, r.z, r.s, 0.f);
    }
    return;
  } else {
    if (wave != 0) return;
    Tri r = part[0];
#pragma unroll
    for (int w = 1; w < NT / kWave; w++) r = tri_merge(r, part[w]);
    if (splits == 1) {
      const float H = finish_entropy(r);
      if (lane == 0) p.H[row] = H;
      detector_push(p, row, H, lane);
      return;
    }
    if (lane == 0)
      reinterpret_cast<float4 *>(p.ws)[(size_t)row * splits + split] = make_float4(r.m, r.z, r.s, 0.f);
  }
}

// The merged triple of a row's split partials ([splits] float4 (m, Z, S, -)
// in the workspace), by one whole wave: each lane loads every 64th partial,
// so the row costs one memory round trip.
__device__ __forceinline__ Tri wave_merge_splits(const EntropyParams &p, int row, int lane) {
  const float4 *q = reinterpret_cast<const float4 *>(p.ws) + (size_t)row * p.splits;
  Tri acc{kNegInf, 0.f, 0.f};
  for (int k = lane; k < p.splits; k += kWave) {
    const float4 v = q[k];
    acc = tri_merge(acc, Tri{v.x, v.y, v.z});
  }
#pragma unroll
  for (int msk = 32; msk >= 1; msk >>= 1) {
    Tri o{shfl_xor(acc.m, msk), shfl_xor(acc.z, msk), shfl_xor(acc.s, msk)};
    acc = tri_merge(acc, o);
  }
  return acc;
}

// Per-row merge of the split partials, then the detector; one wave per
// global row of the batch.
__global__ __launch_bounds__(kWave) void entropy_merge(EntropyBatch b) {
  const int bset = batch_set(b, blockIdx.x);
  const EntropyParams &p = b.set[bset];
  const int row = blockIdx.x - b.row0[bset];
  const int lane = threadIdx.x;
  const float H = finish_entropy(wave_merge_splits(p, row, lane));
  if (lane == 0) p.H[row] = H;
  detector_push(p, row, H, lane);
}

constexpr int kMergeEntries = 1024;  // splits * top_k bound of the sampling merge

// Per-row sampling merge: one wave per row. Entropy and detector as in
// entropy_merge; then the top_k best keys of all splits, the temperature
// softmax over them, the top_p nucleus and the Philox draw. NPL * 64 >=
// splits * top_k.
template <int NPL>
__global__ __launch_bounds__(kWave) void sample_merge(EntropyParams p) {
  const int row = blockIdx.x;
  const int lane = threadIdx.x;
  const int S = p.splits, K = p.top_k;
  const float H = finish_entropy(wave_merge_splits(p, row, lane));
  if (lane == 0) p.H[row] = H;
  detector_push(p, row, H, lane);
  // Candidates.
  const uint64_t *keys = reinterpret_cast<const uint64_t *>(static_cast<const float *>(p.ws) +
                                                            (size_t)p.R * S * 4) + (size_t)row * S * K;
  const int E = S * K;
  uint64_t v[NPL];
#pragma unroll
  for (int i = 0; i < NPL; i++) {
    const int j = lane + i * kWave;
    v[i] = j < E ? keys[j] : 0;
  }
  // The K best keys of all splits, then the draw.
  __shared__ uint64_t win[kTopKMax], sorted[kTopKMax];
  const uint64_t thr = select_threshold<NPL>(v, K, K);
  const int nwin = wave_store_ge<NPL>(win, v, thr, lane);
  sample_draw(p, row, lane, win, sorted, nwin);
}

}  // namespace

static bool row_groups(int R, int V) { return R >= kRowMinRows && V / 8 >= kRowMinVecs; }

static int split_rule(int R, int V) {
  // Enough workgroups to cover the chip (~1024), but at least 1024 vectors of
  // 8 logits per workgroup; and, when the rows alone fill the chip, still no
  // more than one round of the vector loop per workgroup (measured: 256 rows
  // of 152k logits in 8 splits, 2048 workgroups, beat 4 splits by 6%).
  const long nvec = V / 8;
  long s = (1024 + R - 1) / R;
  const long maxs = nvec / 1024 > 0 ? nvec / 1024 : 1;
  if (s > maxs) s = maxs;
  const long one_round = (nvec + kRoundVecs - 1) / kRoundVecs;
  if (s < one_round) s = one_round;
  if (s < 1) s = 1;
  if (s > 1024) s = 1024;
  return (int)s;
}

int entropy_splits(int R, int V) { return row_groups(R, V) ? 1 : split_rule(R, V); }

size_t entropy_workspace_bytes(int R, int V) {
  const int s = entropy_splits(R, V);
  if (s == 1) return 0;
  return (size_t)R * s * 4 * sizeof(float);
}

int sample_splits(int R, int V, int top_k) {
  int s = split_rule(R, V);
  const int maxs = kMergeEntries / (top_k > 0 ? top_k : 1);
  return s < maxs ? s : maxs;
}

size_t sample_workspace_bytes(int R, int V, int top_k) {
  const int s = sample_splits(R, V, top_k);
  return (size_t)R * s * 4 * sizeof(float) + (size_t)R * s * top_k * sizeof(uint64_t);
}

template <typename T, bool VEC>
static void launch_split(const EntropyBatch &b, bool sample, bool rows, dim3 grid, hipStream_t stream) {
  if (sample) hipLaunchKernelGGL((entropy_kernel<T, VEC, true>), grid, dim3(kThreads), 0, stream, b);
  else if (rows) hipLaunchKernelGGL((entropy_kernel<T, VEC, false, kRowThreads>), grid, dim3(kRowThreads), 0, stream, b);
  else hipLaunchKernelGGL((entropy_kernel<T, VEC, false>), grid, dim3(kThreads), 0, stream, b);
}

// The split pass over every row of the batch (one launch), with 16-byte
// loads when every set's rows start 16-byte aligned.
static hipError_t launch_partials(const EntropyBatch &b, bool sample, hipStream_t stream) {
  const EntropyParams &p0 = b.set[0];
  const size_t esz = p0.dtype == 0 ? 4 : 2;
  bool vec = true;
  int vmin = p0.V;
  for (int k = 0; k < b.nsets; k++) {
    vec = vec && ((uintptr_t)b.set[k].logits % 16 == 0) && ((size_t)b.set[k].ld * esz % 16 == 0);
    vmin = b.set[k].V < vmin ? b.set[k].V : vmin;
  }
  const int R = b.row0[b.nsets];
  const bool rows = p0.splits == 1 && row_groups(R, vmin);
  const dim3 grid(p0.splits, R);
  if (p0.dtype == 0) {
    if (vec) launch_split<float, true>(b, sample, rows, grid, stream);
    else launch_split<float, false>(b, sample, rows, grid, stream);
  } else {
    if (vec) launch_split<bf16_t, true>(b, sample, rows, grid, stream);
    else launch_split<bf16_t, false>(b, sample, rows, grid, stream);
  }
  return hipGetLastError();
}

hipError_t entropy_scratch(void **ptr) {
  // Device address of `scratch` on the current device, looked up once per
  // device with that device current (each GPU holds its own copy).
  constexpr int kMaxDevices = 64;
  static std::atomic<void *> cache[kMaxDevices];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void *p = cache[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    cache[dev].store(p, std::memory_order_release);
  }
  *ptr = p;
  return hipSuccess;
}

hipError_t launch_logit_entropy_batch(const EntropyBatch &b, hipStream_t stream) {
  hipError_t e = launch_partials(b, false, stream);
  if (e != hipSuccess || b.set[0].splits == 1) return e;
  hipLaunchKernelGGL(entropy_merge, dim3(b.row0[b.nsets]), dim3(kWave), 0, stream, b);
  return hipGetLastError();
}

hipError_t launch_logit_entropy(const EntropyParams &p, hipStream_t stream) {
  EntropyBatch b{};
  b.set[0] = p;
  b.row0[0] = 0;
  b.row0[1] = p.R;
  b.nsets = 1;
  if (p.top_k <= 0) return launch_logit_entropy_batch(b, stream);
  hipError_t e = launch_partials(b, true, stream);
  if (e != hipSuccess) return e;
  const int E = p.splits * p.top_k;
  if (E <= 64) hipLaunchKernelGGL(sample_merge<1>, dim3(p.R), dim3(kWave), 0, stream, p);
  else if (E <= 128) hipLaunchKernelGGL(sample_merge<2>, dim3(p.R), dim3(kWave), 0, stream, p);
  else if (E <= 256) hipLaunchKernelGGL(sample_merge<4>, dim3(p.R), dim3(kWave), 0, stream, p);
  else if (E <= 512) hipLaunchKernelGGL(sample_merge<8>, dim3(p.R), dim3(kWave), 0, stream, p);
  else hipLaunchKernelGGL(sample_merge<16>, dim3(p.R), dim3(kWave), 0, stream, p);
  return hipGetLastError();
}

}  // namespace kvr
