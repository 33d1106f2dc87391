// Host-side interface between the C ABI layer (api.hip) and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace kvr {

// Geometry and pointers of one kvr_decode_attn call, after validation.
struct AttnParams {
  // own cache [S][L][Hkv][cap][D], pos [S][L][Hkv][cap]
  void *k, *v;
  int32_t *pos;
  int S, L, Hkv, Hq, G, cap, D;
  int dtype;
  // prefix [P][L][Hkv][plen][D]; P == 0 without prefix
  const void *pk, *pv;
  int P, plen, C;  // C = S / P candidates per prefix
  const int32_t *len;
  const void *q;
  const void *k_new, *v_new;
  const int32_t *new_pos;
  void *out;
  float scale;
  // scoring (scores == nullptr: off)
  float *scores;
  int B, W, buffer;
  // split-K partials for the prefix path: ws [nsplit][S][L][Hq] records of
  // 4 + D/2 float slots ((max, sum, -, -) then o / sum as D float16).
  // The context kernel's nwaves waves each take `span` consecutive keys of
  // the flattened (prefix, layer, KV head, key) space; a unit is covered by at
  // most nsplit of them, each leaving one partial record.
  float *ws;
  int nsplit, span, nwaves;
  // The suffix kernel prefetches the first merge_pf pieces of its rows'
  // partials into LDS (merge_blk floats per piece) at wave start.
  int merge_pf, merge_blk;
};

// Work plan of the prefix path (rows = C * G query rows per prefix unit;
// ent_rows = logit rows computed in the context launch, 0 for none);
// identical on the size query and the call. The plan with ent_rows > 0 never
// has more splits than the one without.
void plan_prefix_splits(int D, int P, int L, int Hkv, int plen, int rows, int ent_rows, int *nsplit, int *span,
                        int *nwaves);
size_t attn_workspace_bytes(int S, int L, int Hq, int D, int nsplit);

struct EntropyBatch;
// ent: NULL, or the entropy rows computed in the same launch (rows 16-byte
// aligned, no workspace): with the own-cache kernel, or with a prefix in the
// context kernel (p planned with ent_rows = the batch's rows).
// Context kernels of three and four row blocks (rb = 3 or 4), built in a
// translation unit of their own with the matrix-core accumulators in vector
// registers: the launch, and the waves of it the chip holds at once.
void launch_prefix_wide(int D, int rb, const AttnParams &p, const EntropyBatch *e, hipStream_t stream);
long prefix_slots_wide(int D, int rb, bool rows);
hipError_t launch_decode_attn(const AttnParams &p, const EntropyBatch *ent, hipStream_t stream);

struct ScoreParams {
  const void *k, *v;
  int S, L, Hkv, Hq, G, cap, D, dtype;
  const int32_t *len;
  const void *q_win;
  int nq;
  float scale;
  float *scores;
  int accumulate;
};
hipError_t launch_accumulate_scores(const ScoreParams &p, hipStream_t stream);

struct EvictParams {
  void *k, *v;
  int32_t *pos;
  int S, L, Hkv, cap, D, dtype;
  const int32_t *len;
  int32_t *len_out;  // NULL, or [S] new live lengths
  const float *scores;
  int B, W, buffer;
  int32_t *kept;
};
hipError_t launch_evict_topb(const EvictParams &p, hipStream_t stream);

struct RedundancyParams {
  const void *k;
  int S, L, Hkv, cap, D, dtype;
  const int32_t *len;
  const float *importance;
  float *out;
  int B, W, buffer, pool;
  float lam;
};
size_t redundancy_lds_bytes(int cap, int D);
hipError_t launch_redundancy(const RedundancyParams &p, hipStream_t stream);

struct EntropyParams {
  const void *logits;
  int dtype;
  int R, V;
  int64_t ld;
  float inv_temp;
  float *H;
  float *hist;
  int32_t *cnt;
  uint8_t *flag;
  int window, guard;
  float tau;
  void *ws;
  int splits;
  // Fused sampler (top_k > 0): temperature, top-k, top-p and a Philox draw
  // keyed by (seed, step, row); tokens [R] receive the sampled ids.
  int top_k;
  float inv_t;  // 1 / temperature
  float top_p;
  uint64_t seed, step;
  int32_t *tokens;
};
// Several sets of rows in one launch: global row g belongs to the set k with
// row0[k] <= g < row0[k + 1]. Every set has the same dtype and split count,
// and its ws points at its own R * splits partial records.
constexpr int kEntropyMaxSets = 4;
struct EntropyBatch {
  EntropyParams set[kEntropyMaxSets];
  int row0[kEntropyMaxSets + 1];
  int nsets;
};
int entropy_splits(int R, int V);
size_t entropy_workspace_bytes(int R, int V);
int sample_splits(int R, int V, int top_k);
size_t sample_workspace_bytes(int R, int V, int top_k);
constexpr int kTopKMax = 64;
hipError_t launch_logit_entropy(const EntropyParams &p, hipStream_t stream);
hipError_t launch_logit_entropy_batch(const EntropyBatch &b, hipStream_t stream);
// Library-held device scratch of kvr_logit_entropy_batch_noalloc (split
// partials), per GPU; *ptr receives its address on the current device.
constexpr size_t kEntropyScratchBytes = (size_t)1 << 20;
hipError_t entropy_scratch(void **ptr);

struct ForkParams {
  const void *sk, *sv;
  const int32_t *spos;
  const float *ssc;
  int S_src, cap_src;
  void *dk, *dv;
  int32_t *dpos;
  float *dsc;
  int S_dst, cap_dst;
  int L, Hkv, D, esz;
  int same;  // src and dst are the same cache
  const int32_t *src_index, *len;
};
// Largest L * Hkv and destination count one fork launch covers (its grid
// holds L * Hkv * 2 and S_dst / 8 workgroups in two dimensions).
constexpr long kForkMaxLH = 32767;
constexpr long kForkMaxDst = 65535L * 8;
hipError_t launch_fork(const ForkParams &p, hipStream_t stream);

struct AppendParams {
  void *k, *v;
  int32_t *pos;
  int S, L, Hkv, cap, D, esz;
  const int32_t *len;
  int T;
  const void *k_new, *v_new;
  const int32_t *pos_new;
};
hipError_t launch_append(const AppendParams &p, hipStream_t stream);

}  // namespace kvr
