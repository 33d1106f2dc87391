// C ABI of libkvr: argument validation and dispatch to the gfx950 kernels.
// Every entry point checks its arguments on the host before enqueuing
// anything; on error it returns a status and records a message retrievable
// with kvr_last_error() on the same thread.
#include <hip/hip_runtime.h>

#include <cmath>
#include <stdarg.h>
#include <stdio.h>

#include "../../include/kvr.h"
#include "kvr_internal.h"

namespace {

thread_local char g_err[512] = "";

int fail(int status, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return status;
}

int hip_status(hipError_t e, const char *what) {
  if (e == hipSuccess) return KVR_OK;
  return fail(KVR_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

// Shared checks of a cache description; sets G when Hq > 0.
int check_cache(const kvr_cache *c, int32_t Hq, int *G) {
  if (!c) return fail(KVR_EINVAL, "cache is NULL");
  if (!c->k || !c->v) return fail(KVR_EINVAL, "cache k/v pointer is NULL");
  if (c->S <= 0 || c->L <= 0 || c->Hkv <= 0 || c->cap <= 0 || c->D <= 0)
    return fail(KVR_EINVAL, "cache dims must be positive (S=%d L=%d Hkv=%d cap=%d D=%d)", c->S,
                c->L, c->Hkv, c->cap, c->D);
  if (c->dtype != KVR_F32 && c->dtype != KVR_BF16)
    return fail(KVR_EUNSUPPORTED, "dtype %d is not KVR_F32 or KVR_BF16", c->dtype);
  if (c->D != 64 && c->D != 128) return fail(KVR_EUNSUPPORTED, "head_dim %d is not 64 or 128", c->D);
  if (!aligned16(c->k) || !aligned16(c->v)) return fail(KVR_EINVAL, "cache k/v not 16-byte aligned");
  if ((double)c->S * c->L * c->Hkv > 2147483647.0)
    return fail(KVR_EUNSUPPORTED, "S*L*Hkv exceeds the launch grid");
  if (Hq > 0) {
    if (Hq % c->Hkv != 0) return fail(KVR_EINVAL, "Hq=%d is not a multiple of Hkv=%d", Hq, c->Hkv);
    *G = Hq / c->Hkv;
    if (*G > 16) return fail(KVR_EUNSUPPORTED, "G=%d query heads per KV head exceeds 16", *G);
  }
  return KVR_OK;
}

int check_policy(const kvr_policy *pol, int cap) {
  if (pol->W <= 0 || pol->W >= pol->B)
    return fail(KVR_EINVAL, "policy needs 0 < W < B (B=%d W=%d)", pol->B, pol->W);
  if (pol->buffer < pol->W - 1)
    return fail(KVR_EINVAL, "policy needs buffer >= W-1 (buffer=%d W=%d)", pol->buffer, pol->W);
  if ((long)pol->B + pol->buffer + 1 > cap)
    return fail(KVR_EINVAL, "cap=%d < B+buffer+1=%ld", cap, (long)pol->B + pol->buffer + 1);
  return KVR_OK;
}

}  // namespace

extern "C" {

const char *kvr_strerror(int status) {
  switch (status) {
    case KVR_OK: return "ok";
    case KVR_EINVAL: return "invalid argument";
    case KVR_EUNSUPPORTED: return "unsupported configuration";
    case KVR_EHIP: return "HIP runtime error";
    case KVR_EWORKSPACE: return "workspace missing or too small";
    default: return "unknown status";
  }
}

const char *kvr_last_error(void) { return g_err; }

size_t kvr_decode_attn_workspace_size(const kvr_cache *cache, const kvr_prefix *prefix, int32_t Hq) {
  if (!cache || !prefix || prefix->P <= 0 || cache->dtype != KVR_BF16) return 0;
  if (cache->Hkv <= 0 || Hq <= 0 || Hq % cache->Hkv != 0 || cache->S % prefix->P != 0) return 0;
  int ns = 1, span = 1, nw = 1;
  const int rows = (cache->S / prefix->P) * (Hq / cache->Hkv);
  kvr::plan_prefix_splits(cache->D, prefix->P, cache->L, cache->Hkv, prefix->plen, rows, 0, &ns, &span, &nw);
  return kvr::attn_workspace_bytes(cache->S, cache->L, Hq, cache->D, ns);
}

}  // extern "C"

namespace {

// Validates the arguments of kvr_decode_attn and fills p; ent_rows logit rows
// ride in the same launch (0: none).
int attn_params(const kvr_cache *cache, const kvr_prefix *prefix, const int32_t *len, const void *q, int32_t Hq,
                float scale, const void *k_new, const void *v_new, const int32_t *new_pos, void *out,
                const kvr_policy *policy, float *scores, void *workspace, size_t workspace_bytes, int ent_rows,
                kvr::AttnParams *pp) {
  kvr::AttnParams &p = *pp;
  int G = 0;
  int st = check_cache(cache, Hq, &G);
  if (st) return st;
  if (Hq <= 0) return fail(KVR_EINVAL, "Hq must be positive");
  if (!len || !q || !out) return fail(KVR_EINVAL, "len, q and out are required");
  if (!aligned16(q) || !aligned16(out)) return fail(KVR_EINVAL, "q/out not 16-byte aligned");
  if ((k_new == nullptr) != (v_new == nullptr))
    return fail(KVR_EINVAL, "k_new and v_new must both be given or both be NULL");
  if (k_new && (!aligned16(k_new) || !aligned16(v_new)))
    return fail(KVR_EINVAL, "k_new/v_new not 16-byte aligned");
  if ((policy == nullptr) != (scores == nullptr))
    return fail(KVR_EINVAL, "policy and scores must both be given or both be NULL");
  p = kvr::AttnParams{};
  p.k = cache->k; p.v = cache->v; p.pos = cache->pos;
  p.S = cache->S; p.L = cache->L; p.Hkv = cache->Hkv; p.Hq = Hq; p.G = G;
  p.cap = cache->cap; p.D = cache->D; p.dtype = cache->dtype;
  p.len = len; p.q = q; p.k_new = k_new; p.v_new = v_new; p.new_pos = new_pos; p.out = out;
  p.scale = scale;
  if (policy) {
    st = check_policy(policy, cache->cap);
    if (st) return st;
    if (prefix && prefix->P > 0) return fail(KVR_EINVAL, "scoring is not available with a prefix");
    if (!aligned16(scores)) return fail(KVR_EINVAL, "scores not 16-byte aligned");
    p.scores = scores; p.B = policy->B; p.W = policy->W; p.buffer = policy->buffer;
    if (cache->dtype == KVR_BF16) {
      const size_t lds = ((size_t)G * ((cache->cap + 63) & ~63) + 32) * sizeof(float);
      if (lds > 65536) return fail(KVR_EUNSUPPORTED, "scoring needs %zu bytes of LDS (> 64 KiB)", lds);
    }
  }
  if (prefix && prefix->P > 0) {
    if (!prefix->k || !prefix->v) return fail(KVR_EINVAL, "prefix k/v pointer is NULL");
    if (prefix->plen <= 0) return fail(KVR_EINVAL, "prefix plen must be positive");
    if (cache->S % prefix->P != 0)
      return fail(KVR_EINVAL, "S=%d is not a multiple of the prefix count P=%d", cache->S, prefix->P);
    if (!aligned16(prefix->k) || !aligned16(prefix->v))
      return fail(KVR_EINVAL, "prefix k/v not 16-byte aligned");
    p.pk = prefix->k; p.pv = prefix->v; p.P = prefix->P; p.plen = prefix->plen;
    p.C = cache->S / prefix->P;
    if (cache->dtype == KVR_BF16) {
      if (p.C * G > 64)
        return fail(KVR_EUNSUPPORTED, "%d candidates x %d heads per shared prefix exceeds 64 rows", p.C, G);
      kvr::plan_prefix_splits(p.D, p.P, p.L, p.Hkv, p.plen, p.C * G, ent_rows, &p.nsplit, &p.span, &p.nwaves);
      const size_t need = kvr::attn_workspace_bytes(p.S, p.L, Hq, p.D, p.nsplit);
      if (!workspace || workspace_bytes < need)
        return fail(KVR_EWORKSPACE, "workspace of %zu bytes needed, %zu given", need, workspace_bytes);
      if (!aligned16(workspace)) return fail(KVR_EINVAL, "workspace not 16-byte aligned");
      p.ws = static_cast<float *>(workspace);
    }
  }
  if (cache->dtype == KVR_F32) {
    const size_t nt = (size_t)(p.P > 0 ? p.plen : 0) + p.cap;
    const size_t lds = ((size_t)G * p.D + (size_t)G * nt + 32) * sizeof(float);
    if (lds > 65536) return fail(KVR_EUNSUPPORTED, "float32 path needs %zu bytes of LDS (> 64 KiB)", lds);
  }
  return KVR_OK;
}

}  // namespace

extern "C" {

int kvr_decode_attn(const kvr_cache *cache, const kvr_prefix *prefix, const int32_t *len,
                    const void *q, int32_t Hq, float scale, const void *k_new, const void *v_new,
                    const int32_t *new_pos, void *out, const kvr_policy *policy, float *scores,
                    void *workspace, size_t workspace_bytes, hipStream_t stream) {
  kvr::AttnParams p;
  const int st = attn_params(cache, prefix, len, q, Hq, scale, k_new, v_new, new_pos, out, policy, scores,
                             workspace, workspace_bytes, 0, &p);
  if (st) return st;
  return hip_status(kvr::launch_decode_attn(p, nullptr, stream), "kvr_decode_attn launch");
}

int kvr_accumulate_scores(const kvr_cache *cache, const int32_t *len, const void *q_win,
                          int32_t nq, int32_t Hq, float scale, float *scores, int32_t accumulate,
                          hipStream_t stream) {
  int G = 0;
  int st = check_cache(cache, Hq, &G);
  if (st) return st;
  if (Hq <= 0 || nq <= 0) return fail(KVR_EINVAL, "Hq and nq must be positive");
  if (!len || !q_win || !scores) return fail(KVR_EINVAL, "len, q_win and scores are required");
  const size_t lds = cache->dtype == KVR_BF16
                        ? (size_t)cache->cap * sizeof(unsigned long long)
                        : ((size_t)cache->D + 2 * (size_t)cache->cap) * sizeof(float);
  if (lds > 65536) return fail(KVR_EUNSUPPORTED, "cap=%d needs too much LDS", cache->cap);
  if (!aligned16(q_win)) return fail(KVR_EINVAL, "q_win not 16-byte aligned");
  if ((double)G * nq * cache->D * 4 >= 2147483647.0)
    return fail(KVR_EUNSUPPORTED, "window of %d rows is too large", G * nq);
  kvr::ScoreParams p{};
  p.k = cache->k; p.v = cache->v;
  p.S = cache->S; p.L = cache->L; p.Hkv = cache->Hkv; p.Hq = Hq; p.G = G;
  p.cap = cache->cap; p.D = cache->D; p.dtype = cache->dtype;
  p.len = len; p.q_win = q_win; p.nq = nq; p.scale = scale; p.scores = scores;
  p.accumulate = accumulate != 0;
  return hip_status(kvr::launch_accumulate_scores(p, stream), "kvr_accumulate_scores launch");
}

int kvr_evict_topb(const kvr_cache *cache, const int32_t *len, int32_t *len_out, const float *scores,
                   const kvr_policy *policy, int32_t *kept, hipStream_t stream) {
  int G = 0;
  int st = check_cache(cache, 0, &G);
  if (st) return st;
  if (!len || !scores || !policy) return fail(KVR_EINVAL, "len, scores and policy are required");
  if (len_out) {
    const char *a = reinterpret_cast<const char *>(len), *b = reinterpret_cast<const char *>(len_out);
    const size_t n = (size_t)cache->S * sizeof(int32_t);
    if (a < b + n && b < a + n) return fail(KVR_EINVAL, "len_out overlaps len");
  }
  st = check_policy(policy, cache->cap);
  if (st) return st;
  const size_t lds = (size_t)(cache->cap + policy->B) * sizeof(uint32_t);
  if (lds > 65536) return fail(KVR_EUNSUPPORTED, "cap=%d needs too much LDS", cache->cap);
  kvr::EvictParams p{};
  p.k = cache->k; p.v = cache->v; p.pos = cache->pos;
  p.S = cache->S; p.L = cache->L; p.Hkv = cache->Hkv; p.cap = cache->cap; p.D = cache->D;
  p.dtype = cache->dtype; p.len = len; p.len_out = len_out; p.scores = scores;
  p.B = policy->B; p.W = policy->W; p.buffer = policy->buffer; p.kept = kept;
  return hip_status(kvr::launch_evict_topb(p, stream), "kvr_evict_topb launch");
}

int kvr_redundancy_scores(const kvr_cache *cache, const int32_t *len, const float *importance,
                          const kvr_policy *policy, float lam, int32_t pool, float *out,
                          hipStream_t stream) {
  int G = 0;
  int st = check_cache(cache, 0, &G);
  if (st) return st;
  if (!len || !importance || !out || !policy)
    return fail(KVR_EINVAL, "len, importance, policy and out are required");
  st = check_policy(policy, cache->cap);
  if (st) return st;
  if (!(lam >= 0.f && lam <= 1.f)) return fail(KVR_EINVAL, "lambda must lie in [0, 1]");
  if (pool < 1) return fail(KVR_EINVAL, "pool=%d must be at least 1", pool);
  const size_t lds = kvr::redundancy_lds_bytes(cache->cap, cache->D);
  if (lds > 65536) return fail(KVR_EUNSUPPORTED, "cap=%d needs %zu bytes of LDS (> 64 KiB)", cache->cap, lds);
  kvr::RedundancyParams p{};
  p.k = cache->k; p.S = cache->S; p.L = cache->L; p.Hkv = cache->Hkv; p.cap = cache->cap;
  p.D = cache->D; p.dtype = cache->dtype; p.len = len; p.importance = importance; p.out = out;
  p.B = policy->B; p.W = policy->W; p.buffer = policy->buffer; p.pool = pool; p.lam = lam;
  return hip_status(kvr::launch_redundancy(p, stream), "kvr_redundancy_scores launch");
}

int kvr_fork(const kvr_cache *src, const kvr_cache *dst, const int32_t *src_index,
             const int32_t *len, const float *src_scores, float *dst_scores,
             hipStream_t stream) {
  int G = 0;
  int st = check_cache(src, 0, &G);
  if (st) return st;
  st = check_cache(dst, 0, &G);
  if (st) return st;
  if (src->L != dst->L || src->Hkv != dst->Hkv || src->D != dst->D || src->dtype != dst->dtype)
    return fail(KVR_EINVAL, "src and dst caches differ in L, Hkv, D or dtype");
  if (!src_index || !len) return fail(KVR_EINVAL, "src_index and len are required");
  if ((src_scores == nullptr) != (dst_scores == nullptr))
    return fail(KVR_EINVAL, "src_scores and dst_scores must both be given or both be NULL");
  if (dst->pos && !src->pos) return fail(KVR_EINVAL, "dst tracks positions but src does not");
  const bool same = src->k == dst->k;
  if (same && (src->v != dst->v || src->S != dst->S || src->cap != dst->cap ||
               src->pos != dst->pos || src_scores != dst_scores))
    return fail(KVR_EINVAL, "src and dst share k but are not the same cache");
  if (!same && (src->v == dst->v))
    return fail(KVR_EINVAL, "src and dst share v but not k");
  if ((long)dst->L * dst->Hkv > kvr::kForkMaxLH || dst->S > kvr::kForkMaxDst)
    return fail(KVR_EUNSUPPORTED, "fork of L*Hkv=%ld units over S=%d destinations (at most %ld and %ld)",
                (long)dst->L * dst->Hkv, dst->S, kvr::kForkMaxLH, kvr::kForkMaxDst);
  kvr::ForkParams p{};
  p.sk = src->k; p.sv = src->v; p.spos = dst->pos ? src->pos : nullptr; p.ssc = src_scores;
  p.S_src = src->S; p.cap_src = src->cap;
  p.dk = dst->k; p.dv = dst->v; p.dpos = dst->pos; p.dsc = dst_scores;
  p.S_dst = dst->S; p.cap_dst = dst->cap;
  p.L = dst->L; p.Hkv = dst->Hkv; p.D = dst->D; p.esz = dst->dtype == KVR_F32 ? 4 : 2;
  p.same = same; p.src_index = src_index; p.len = len;
  return hip_status(kvr::launch_fork(p, stream), "kvr_fork launch");
}

int kvr_append(const kvr_cache *cache, const int32_t *len, int32_t T, const void *k_new,
               const void *v_new, const int32_t *pos_new, hipStream_t stream) {
  int G = 0;
  int st = check_cache(cache, 0, &G);
  if (st) return st;
  if (T < 0) return fail(KVR_EINVAL, "T=%d is negative", T);
  if (pos_new && !cache->pos) return fail(KVR_EINVAL, "pos_new given but the cache has no pos");
  if (T == 0) return KVR_OK;
  if (!len || !k_new || !v_new) return fail(KVR_EINVAL, "len, k_new and v_new are required");
  if (!aligned16(k_new) || !aligned16(v_new)) return fail(KVR_EINVAL, "k_new/v_new not 16-byte aligned");
  const int esz = cache->dtype == KVR_F32 ? 4 : 2;
  const long chunks = ((long)T * cache->D * esz / 16 + 1023) / 1024;
  if (chunks > 65535) return fail(KVR_EUNSUPPORTED, "T=%d tokens per call is too many", T);
  kvr::AppendParams p{};
  p.k = cache->k; p.v = cache->v; p.pos = cache->pos;
  p.S = cache->S; p.L = cache->L; p.Hkv = cache->Hkv; p.cap = cache->cap; p.D = cache->D;
  p.esz = esz; p.len = len; p.T = T; p.k_new = k_new; p.v_new = v_new; p.pos_new = pos_new;
  return hip_status(kvr::launch_append(p, stream), "kvr_append launch");
}

size_t kvr_logit_entropy_workspace_size(int32_t R, int32_t V) {
  if (R <= 0 || V <= 0) return 0;
  return kvr::entropy_workspace_bytes(R, V);
}

}  // extern "C"

namespace {

// Checks shared by the entropy entry points; fills everything but splits/ws.
int entropy_params(const void *logits, int32_t dtype, int32_t R, int32_t V, int64_t ld,
                   float inv_temp, float *H, const kvr_detector *det, kvr::EntropyParams *p) {
  if (!logits || !H) return fail(KVR_EINVAL, "logits and H are required");
  if (dtype != KVR_F32 && dtype != KVR_BF16) return fail(KVR_EUNSUPPORTED, "dtype %d", dtype);
  if (R <= 0 || V <= 0 || ld < V) return fail(KVR_EINVAL, "need R > 0, V > 0, ld >= V (R=%d V=%d ld=%ld)", R, V, (long)ld);
  if (R > 65535) return fail(KVR_EUNSUPPORTED, "R=%d rows exceeds 65535", R);
  if (!(inv_temp > 0.f) || !std::isfinite(inv_temp))
    return fail(KVR_EINVAL, "inv_temp must be positive and finite (got %g)", (double)inv_temp);
  *p = kvr::EntropyParams{};
  p->logits = logits; p->dtype = dtype; p->R = R; p->V = V; p->ld = ld; p->inv_temp = inv_temp; p->H = H;
  if (det) {
    if (!det->hist || !det->cnt || !det->flag) return fail(KVR_EINVAL, "detector arrays are required");
    if (det->window <= 0 || det->guard < 0) return fail(KVR_EINVAL, "detector window must be positive");
    p->hist = det->hist; p->cnt = det->cnt; p->flag = det->flag;
    p->window = det->window; p->guard = det->guard; p->tau = det->tau;
  }
  return KVR_OK;
}

int attach_workspace(kvr::EntropyParams *p, size_t need, void *workspace, size_t workspace_bytes) {
  if (need == 0) return KVR_OK;
  if (!workspace || workspace_bytes < need)
    return fail(KVR_EWORKSPACE, "workspace of %zu bytes needed, %zu given", need, workspace_bytes);
  if (!aligned16(workspace)) return fail(KVR_EINVAL, "workspace not 16-byte aligned");
  p->ws = workspace;
  return KVR_OK;
}

}  // namespace

extern "C" {

int kvr_logit_entropy(const void *logits, int32_t dtype, int32_t R, int32_t V, int64_t ld,
                      float inv_temp, float *H, const kvr_detector *det, void *workspace,
                      size_t workspace_bytes, hipStream_t stream) {
  kvr::EntropyParams p;
  int st = entropy_params(logits, dtype, R, V, ld, inv_temp, H, det, &p);
  if (st) return st;
  p.splits = kvr::entropy_splits(R, V);
  st = attach_workspace(&p, kvr::entropy_workspace_bytes(R, V), workspace, workspace_bytes);
  if (st) return st;
  return hip_status(kvr::launch_logit_entropy(p, stream), "kvr_logit_entropy launch");
}

}  // extern "C"

namespace {

// Validates a batch and fills b (all but the workspace pointers); *need gets
// the workspace size. With shapes_only, the sets' pointers are not checked
// (the workspace size depends on the shapes alone).
int check_sampler(const kvr_sampler *sampler) {
  if (!(sampler->temperature > 0.f)) return fail(KVR_EINVAL, "temperature must be positive");
  if (sampler->top_k < 1 || sampler->top_k > kvr::kTopKMax)
    return fail(KVR_EINVAL, "top_k=%d is outside 1..%d", sampler->top_k, kvr::kTopKMax);
  if (!(sampler->top_p > 0.f && sampler->top_p <= 1.f)) return fail(KVR_EINVAL, "top_p must lie in (0, 1]");
  return KVR_OK;
}

int entropy_batch(const kvr_logit_set *sets, int32_t nsets, kvr::EntropyBatch *b, size_t *need,
                  bool shapes_only = false) {
  if (!sets) return fail(KVR_EINVAL, "sets is required");
  if (nsets < 1 || nsets > kvr::kEntropyMaxSets)
    return fail(KVR_EINVAL, "nsets=%d outside 1..%d", nsets, kvr::kEntropyMaxSets);
  *b = kvr::EntropyBatch{};
  b->nsets = nsets;
  long rows = 0;
  int vmin = 0;
  for (int k = 0; k < nsets; k++) {
    const kvr_logit_set &s = sets[k];
    const void *any = reinterpret_cast<const void *>(16);
    int st = shapes_only ? entropy_params(any, s.dtype, s.R, s.V, s.ld, s.inv_temp, (float *)any, nullptr, &b->set[k])
                         : entropy_params(s.logits, s.dtype, s.R, s.V, s.ld, s.inv_temp, s.H, s.det, &b->set[k]);
    if (st) return st;
    if (s.dtype != sets[0].dtype) return fail(KVR_EINVAL, "set %d dtype %d differs from set 0's %d", k, s.dtype, sets[0].dtype);
    b->row0[k] = (int)rows;
    rows += s.R;
    if (rows > 65535) return fail(KVR_EINVAL, "%ld rows in the batch exceeds 65535", rows);
    vmin = k == 0 || s.V < vmin ? s.V : vmin;
  }
  b->row0[nsets] = (int)rows;
  const int splits = kvr::entropy_splits((int)rows, vmin);
  for (int k = 0; k < nsets; k++) b->set[k].splits = splits;
  *need = splits == 1 ? 0 : (size_t)rows * splits * 4 * sizeof(float);
  return KVR_OK;
}

}  // namespace

extern "C" {

size_t kvr_logit_entropy_batch_workspace_size(const kvr_logit_set *sets, int32_t nsets) {
  kvr::EntropyBatch b;
  size_t need = 0;
  if (entropy_batch(sets, nsets, &b, &need, true)) return 0;
  return need;
}

int kvr_logit_entropy_batch(const kvr_logit_set *sets, int32_t nsets, void *workspace,
                            size_t workspace_bytes, hipStream_t stream) {
  kvr::EntropyBatch b;
  size_t need = 0;
  int st = entropy_batch(sets, nsets, &b, &need);
  if (st) return st;
  if (need) {
    if (!workspace || workspace_bytes < need)
      return fail(KVR_EWORKSPACE, "workspace of %zu bytes needed, %zu given", need, workspace_bytes);
    if (!aligned16(workspace)) return fail(KVR_EINVAL, "workspace not 16-byte aligned");
    for (int k = 0; k < nsets; k++)
      b.set[k].ws = static_cast<char *>(workspace) + (size_t)b.row0[k] * b.set[k].splits * 4 * sizeof(float);
  }
  return hip_status(kvr::launch_logit_entropy_batch(b, stream), "kvr_logit_entropy_batch launch");
}

int kvr_logit_entropy_batch_noalloc(const kvr_logit_set *sets, int32_t nsets, hipStream_t stream) {
  kvr::EntropyBatch b;
  size_t need = 0;
  int st = entropy_batch(sets, nsets, &b, &need);
  if (st) return st;
  if (need > kvr::kEntropyScratchBytes)
    return fail(KVR_EUNSUPPORTED, "the split partials need %zu bytes, more than the %zu bytes of library scratch",
                need, kvr::kEntropyScratchBytes);
  if (need) {
    int dev = -1, sdev = -1;
    st = hip_status(hipGetDevice(&dev), "kvr_logit_entropy_batch_noalloc: hipGetDevice");
    if (st) return st;
    st = hip_status(hipStreamGetDevice(stream, &sdev), "kvr_logit_entropy_batch_noalloc: hipStreamGetDevice");
    if (st) return st;
    if (sdev != dev)
      return fail(KVR_EINVAL, "stream belongs to device %d, the current device is %d", sdev, dev);
    void *ws = nullptr;
    st = hip_status(kvr::entropy_scratch(&ws), "kvr_logit_entropy_batch_noalloc: scratch address");
    if (st) return st;
    for (int k = 0; k < nsets; k++)
      b.set[k].ws = static_cast<char *>(ws) + (size_t)b.row0[k] * b.set[k].splits * 4 * sizeof(float);
  }
  return hip_status(kvr::launch_logit_entropy_batch(b, stream), "kvr_logit_entropy_batch_noalloc launch");
}

size_t kvr_logit_entropy_sample_workspace_size(int32_t R, int32_t V, int32_t top_k) {
  if (R <= 0 || V <= 0 || top_k < 1 || top_k > kvr::kTopKMax) return 0;
  return kvr::sample_workspace_bytes(R, V, top_k);
}

int kvr_logit_entropy_sample(const void *logits, int32_t dtype, int32_t R, int32_t V, int64_t ld,
                             float inv_temp, float *H, const kvr_detector *det,
                             const kvr_sampler *sampler, int32_t *tokens, void *workspace,
                             size_t workspace_bytes, hipStream_t stream) {
  kvr::EntropyParams p;
  int st = entropy_params(logits, dtype, R, V, ld, inv_temp, H, det, &p);
  if (st) return st;
  if (!sampler || !tokens) return fail(KVR_EINVAL, "sampler and tokens are required");
  st = check_sampler(sampler);
  if (st) return st;
  p.top_k = sampler->top_k;
  p.inv_t = 1.0f / sampler->temperature;
  p.top_p = sampler->top_p;
  p.seed = sampler->seed;
  p.step = sampler->step;
  p.tokens = tokens;
  p.splits = kvr::sample_splits(R, V, sampler->top_k);
  st = attach_workspace(&p, kvr::sample_workspace_bytes(R, V, sampler->top_k), workspace, workspace_bytes);
  if (st) return st;
  return hip_status(kvr::launch_logit_entropy(p, stream), "kvr_logit_entropy_sample launch");
}

}  // extern "C"

namespace {

// Validates the arguments of the fused attention + entropy calls and fills p
// and b (the sampler, when given, applies to every set).
int fused_params(const kvr_cache *cache, const kvr_prefix *prefix, const int32_t *len, const void *q, int32_t Hq,
                 float scale, const void *k_new, const void *v_new, const int32_t *new_pos, void *out,
                 const kvr_policy *policy, float *scores, void *workspace, size_t workspace_bytes,
                 const kvr_logit_set *sets, int32_t nsets, const kvr_sampler *sampler, int32_t *const *tokens,
                 kvr::AttnParams *p, kvr::EntropyBatch *b) {
  size_t need = 0;
  int st = entropy_batch(sets, nsets, b, &need);
  if (st) return st;
  st = attn_params(cache, prefix, len, q, Hq, scale, k_new, v_new, new_pos, out, policy, scores, workspace,
                   workspace_bytes, b->row0[nsets], p);
  if (st) return st;
  const size_t esz = sets[0].dtype == KVR_F32 ? 4 : 2;
  for (int k = 0; k < nsets; k++)
    if (!aligned16(sets[k].logits) || ((size_t)sets[k].ld * esz) % 16 != 0)
      return fail(KVR_EINVAL, "set %d: logit rows must start 16-byte aligned (logits and ld * element size)", k);
  if ((double)b->row0[nsets] + (double)cache->S * cache->L * cache->Hkv > 2147483647.0)
    return fail(KVR_EUNSUPPORTED, "logit rows plus attention units exceed the launch grid");
  if (sampler) {
    st = check_sampler(sampler);
    if (st) return st;
    if (!tokens) return fail(KVR_EINVAL, "tokens is required with a sampler");
    for (int k = 0; k < nsets; k++) {
      if (!tokens[k]) return fail(KVR_EINVAL, "set %d: tokens pointer is NULL", k);
      kvr::EntropyParams &e = b->set[k];
      e.top_k = sampler->top_k;
      e.inv_t = 1.0f / sampler->temperature;
      e.top_p = sampler->top_p;
      e.seed = sampler->seed;
      e.step = sampler->step;
      e.tokens = tokens[k];
    }
  }
  return KVR_OK;
}

}  // namespace

extern "C" {

int kvr_decode_attn_entropy(const kvr_cache *cache, const kvr_prefix *prefix, const int32_t *len, const void *q,
                            int32_t Hq, float scale, const void *k_new, const void *v_new, const int32_t *new_pos,
                            void *out, const kvr_policy *policy, float *scores, void *workspace,
                            size_t workspace_bytes, const kvr_logit_set *sets, int32_t nsets, hipStream_t stream) {
  kvr::AttnParams p;
  kvr::EntropyBatch b;
  const int st = fused_params(cache, prefix, len, q, Hq, scale, k_new, v_new, new_pos, out, policy, scores,
                              workspace, workspace_bytes, sets, nsets, nullptr, nullptr, &p, &b);
  if (st) return st;
  return hip_status(kvr::launch_decode_attn(p, &b, stream), "kvr_decode_attn_entropy launch");
}

int kvr_decode_attn_entropy_sample(const kvr_cache *cache, const kvr_prefix *prefix, const int32_t *len,
                                   const void *q, int32_t Hq, float scale, const void *k_new, const void *v_new,
                                   const int32_t *new_pos, void *out, const kvr_policy *policy, float *scores,
                                   void *workspace, size_t workspace_bytes, const kvr_logit_set *sets,
                                   int32_t nsets, const kvr_sampler *sampler, int32_t *const *tokens,
                                   hipStream_t stream) {
  if (!sampler) return fail(KVR_EINVAL, "sampler is required");
  kvr::AttnParams p;
  kvr::EntropyBatch b;
  const int st = fused_params(cache, prefix, len, q, Hq, scale, k_new, v_new, new_pos, out, policy, scores,
                              workspace, workspace_bytes, sets, nsets, sampler, tokens, &p, &b);
  if (st) return st;
  return hip_status(kvr::launch_decode_attn(p, &b, stream), "kvr_decode_attn_entropy_sample launch");
}

}  // extern "C"
