// C ABI of the XAttention library: argument validation, workspace sizing and
// the stream-ordered launch sequence. Declarations and the contract of every
// entry point are in include/xattn.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "xattn.h"
#include "common.h"

namespace xattn_host {

thread_local char g_err[512] = "";

// Records the message of a failing call (read back by xattn_last_error).
int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

}  // namespace xattn_host

namespace {

using xattn_host::fail;
using xattn_host::g_err;

int ok() {
  g_err[0] = '\0';
  return XATTN_OK;
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

int check_dims(const xattn_dims* d, XattnShape* s) {
  if (!d) return fail(XATTN_ERR_ARG, "dims is NULL");
  if (d->batch < 1 || d->hq < 1 || d->hkv < 1 || d->seq < 1 || d->head_dim < 1)
    return fail(XATTN_ERR_ARG, "dims must be positive (batch=%d hq=%d hkv=%d seq=%d d=%d)",
                d->batch, d->hq, d->hkv, d->seq, d->head_dim);
  if (d->hq % d->hkv != 0)
    return fail(XATTN_ERR_ARG, "hq (%d) must be a multiple of hkv (%d)", d->hq, d->hkv);
  if (d->causal != 0 && d->causal != 1)
    return fail(XATTN_ERR_ARG, "causal must be 0 or 1 (got %d)", d->causal);
  if (d->seq % xattn::kBlock != 0)
    return fail(XATTN_ERR_ARG, "seq (%d) must be a multiple of the block size %d", d->seq,
                xattn::kBlock);
  if (d->head_dim != xattn::kHeadDim)
    return fail(XATTN_ERR_UNSUPPORTED, "head_dim %d not supported (only %d)", d->head_dim,
                xattn::kHeadDim);
  if (d->seq / xattn::kBlock > 2048)
    return fail(XATTN_ERR_UNSUPPORTED, "seq %d exceeds 262144 (2048 blocks)", d->seq);
  const long long elems = (long long)d->batch * d->hq * d->seq * d->head_dim;
  if (elems > (1ll << 40)) return fail(XATTN_ERR_UNSUPPORTED, "problem too large");
  *s = XattnShape{d->batch, d->hq, d->hkv, d->seq, d->head_dim, d->causal};
  return XATTN_OK;
}

int check_block(int block) {
  if (block <= 0) return fail(XATTN_ERR_ARG, "block must be positive (got %d)", block);
  if (block != xattn::kBlock)
    return fail(XATTN_ERR_UNSUPPORTED, "block %d not supported (only %d)", block, xattn::kBlock);
  return XATTN_OK;
}

int check_stride(int stride) {
  if (stride <= 0 || xattn::kBlock % stride != 0)
    return fail(XATTN_ERR_ARG, "stride %d must be a positive divisor of the block size", stride);
  if (stride > 64) return fail(XATTN_ERR_UNSUPPORTED, "stride %d not supported (<= 64)", stride);
  return XATTN_OK;
}

int check_tau(float tau) {
  if (!(tau > 0.f)) return fail(XATTN_ERR_ARG, "tau must be > 0 (got %g)", (double)tau);
  return XATTN_OK;
}

int hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess)
    return fail(XATTN_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

SelectParams uniform_threshold(const XattnShape& s, float tau) {
  SelectParams p{};
  p.mode = kSelectThreshold;
  p.hq = s.hq;
  p.uniform = 1;
  p.v[0] = tau;
  return p;
}

SelectParams per_head(const XattnShape& s, int mode) {
  SelectParams p{};
  p.mode = mode;
  p.hq = s.hq;
  p.uniform = 0;
  return p;
}

int check_heads(const XattnShape& s, const void* values) {
  if (!values) return fail(XATTN_ERR_ARG, "the per-head parameter array is NULL");
  if (s.hq > kMaxSelectHeads)
    return fail(XATTN_ERR_UNSUPPORTED, "per-head selection supports hq <= %d (got %d)",
                kMaxSelectHeads, s.hq);
  return XATTN_OK;
}

size_t scores_bytes(const XattnShape& s) { return (size_t)s.HQ() * s.NB() * s.NB() * 4; }
size_t idx_bytes(const XattnShape& s) { return (size_t)s.HQ() * s.NB() * s.NB() * 4; }
size_t cnt_bytes(const XattnShape& s) { return (size_t)s.HQ() * s.NB() * 4; }

}  // namespace

extern "C" {

int xattn_score_workspace_size(const xattn_dims* dims, int block, int stride, size_t* bytes) {
  XattnShape s;
  int rc;
  if ((rc = check_dims(dims, &s)) || (rc = check_block(block)) || (rc = check_stride(stride)))
    return rc;
  if (!bytes) return fail(XATTN_ERR_ARG, "bytes is NULL");
  *bytes = score_scratch_bytes(s, stride);
  return ok();
}

int xattn_score(const void* q, const void* k, const xattn_dims* dims, int block, int stride,
                float* scores, void* workspace, size_t workspace_bytes, void* stream) {
  XattnShape s;
  int rc;
  if ((rc = check_dims(dims, &s)) || (rc = check_block(block)) || (rc = check_stride(stride)))
    return rc;
  if (!q || !k || !scores) return fail(XATTN_ERR_ARG, "q, k and scores must be non-NULL");
  const size_t need = score_scratch_bytes(s, stride);
  if (!workspace || workspace_bytes < need)
    return fail(XATTN_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                workspace ? workspace_bytes : (size_t)0);
  return hip_status(launch_score(q, k, s, stride, nullptr, scores, workspace,
                                  (hipStream_t)stream),
                    "xattn_score launch");
}

int xattn_score_pattern(const void* q, const void* k, const xattn_dims* dims, int block,
                        int stride, const int32_t* qsub, float* scores, void* workspace,
                        size_t workspace_bytes, void* stream) {
  XattnShape s;
  int rc;
  if ((rc = check_dims(dims, &s)) || (rc = check_block(block)) || (rc = check_stride(stride)))
    return rc;
  if (!qsub) return fail(XATTN_ERR_ARG, "qsub is NULL");
  bool seen[64] = {};
  for (int t = 0; t < stride; ++t) {
    if (qsub[t] < 0 || qsub[t] >= stride || seen[qsub[t]])
      return fail(XATTN_ERR_ARG, "qsub must be a permutation of 0..%d (qsub[%d] = %d)",
                  stride - 1, t, qsub[t]);
    seen[qsub[t]] = true;
  }
  if (!q || !k || !scores) return fail(XATTN_ERR_ARG, "q, k and scores must be non-NULL");
  const size_t need = score_scratch_bytes(s, stride);
  if (!workspace || workspace_bytes < need)
    return fail(XATTN_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                workspace ? workspace_bytes : (size_t)0);
  return hip_status(launch_score(q, k, s, stride, qsub, scores, workspace, (hipStream_t)stream),
                    "xattn_score_pattern launch");
}

int xattn_select(const float* scores, const xattn_dims* dims, int block, float tau,
                 int32_t* idx, int32_t* cnt, void* stream) {
  XattnShape s;
  int rc;
  if ((rc = check_dims(dims, &s)) || (rc = check_block(block)) || (rc = check_tau(tau)))
    return rc;
  if (!scores || !idx || !cnt) return fail(XATTN_ERR_ARG, "scores, idx and cnt must be non-NULL");
  return hip_status(launch_select(scores, s, uniform_threshold(s, tau), idx, cnt,
                                  (hipStream_t)stream),
                    "xattn_select launch");
}

int xattn_select_heads(const float* scores, const xattn_dims* dims, int block,
                       const float* tau_h, int32_t* idx, int32_t* cnt, void* stream) {
  XattnShape s;
  int rc;
  if ((rc = check_dims(dims, &s)) || (rc = check_block(block)) || (rc = check_heads(s, tau_h)))
    return rc;
  SelectParams p = per_head(s, kSelectThreshold);
  for (int i = 0; i < s.hq; ++i) {
    if (!(tau_h[i] > 0.f))
      return fail(XATTN_ERR_ARG, "tau_h[%d] must be > 0 (got %g)", i, (double)tau_h[i]);
    p.v[i] = tau_h[i];
  }
  if (!scores || !idx || !cnt) return fail(XATTN_ERR_ARG, "scores, idx and cnt must be non-NULL");
  return hip_status(launch_select(scores, s, p, idx, cnt, (hipStream_t)stream),
                    "xattn_select_heads launch");
}

int xattn_select_topk(const float* scores, const xattn_dims* dims, int block,
                      const int32_t* k_h, int32_t* idx, int32_t* cnt, void* stream) {
  XattnShape s;
  int rc;
  if ((rc = check_dims(dims, &s)) || (rc = check_block(block)) || (rc = check_heads(s, k_h)))
    return rc;
  SelectParams p = per_head(s, kSelectTopK);
  for (int i = 0; i < s.hq; ++i) {
    if (k_h[i] < 1) return fail(XATTN_ERR_ARG, "k_h[%d] must be >= 1 (got %d)", i, k_h[i]);
    p.k[i] = k_h[i];
  }
  if (!scores || !idx || !cnt) return fail(XATTN_ERR_ARG, "scores, idx and cnt must be non-NULL");
  return hip_status(launch_select(scores, s, p, idx, cnt, (hipStream_t)stream),
                    "xattn_select_topk launch");
}

int xattn_select_ratio(const float* scores, const xattn_dims* dims, int block,
                       const float* ratio_h, int32_t* idx, int32_t* cnt, void* stream) {
  XattnShape s;
  int rc;
  if ((rc = check_dims(dims, &s)) || (rc = check_block(block)) || (rc = check_heads(s, ratio_h)))
    return rc;
  SelectParams p = per_head(s, kSelectRatio);
  for (int i = 0; i < s.hq; ++i) {
    const float r = ratio_h[i];
    if (!(r > 0.f) || !std::isfinite(r))
      return fail(XATTN_ERR_ARG, "ratio_h[%d] must be finite and > 0 (got %g)", i, (double)r);
    p.v[i] = r;
  }
  if (!scores || !idx || !cnt) return fail(XATTN_ERR_ARG, "scores, idx and cnt must be non-NULL");
  return hip_status(launch_select(scores, s, p, idx, cnt, (hipStream_t)stream),
                    "xattn_select_ratio launch");
}

int xattn_block_sparse_attn(const void* q, const void* k, const void* v, const xattn_dims* dims,
                            int block, const int32_t* idx, const int32_t* cnt, void* o,
                            float* lse, void* stream) {
  XattnShape s;
  int rc;
  if ((rc = check_dims(dims, &s)) || (rc = check_block(block))) return rc;
  if (!q || !k || !v || !idx || !cnt || !o)
    return fail(XATTN_ERR_ARG, "q, k, v, idx, cnt and o must be non-NULL");
  return hip_status(launch_attn(q, k, v, s, idx, cnt, false, o, lse, (hipStream_t)stream),
                    "xattn_block_sparse_attn launch");
}

int xattn_dense_attn(const void* q, const void* k, const void* v, const xattn_dims* dims,
                     void* o, float* lse, void* stream) {
  XattnShape s;
  int rc;
  if ((rc = check_dims(dims, &s))) return rc;
  if (!q || !k || !v || !o) return fail(XATTN_ERR_ARG, "q, k, v and o must be non-NULL");
  return hip_status(launch_attn(q, k, v, s, nullptr, nullptr, true, o, lse, (hipStream_t)stream),
                    "xattn_dense_attn launch");
}

int xattn_forward_layout(const xattn_dims* dims, int block, int stride, size_t* scores_off,
                         size_t* idx_off, size_t* cnt_off, size_t* scratch_off) {
  XattnShape s;
  int rc;
  if ((rc = check_dims(dims, &s)) || (rc = check_block(block)) || (rc = check_stride(stride)))
    return rc;
  const size_t o_sc = 0;
  const size_t o_idx = align_up(o_sc + scores_bytes(s));
  const size_t o_cnt = align_up(o_idx + idx_bytes(s));
  const size_t o_scr = align_up(o_cnt + cnt_bytes(s));
  if (scores_off) *scores_off = o_sc;
  if (idx_off) *idx_off = o_idx;
  if (cnt_off) *cnt_off = o_cnt;
  if (scratch_off) *scratch_off = o_scr;
  return ok();
}

int xattn_forward_workspace_size(const xattn_dims* dims, int block, int stride, size_t* bytes) {
  size_t scr = 0;
  int rc = xattn_forward_layout(dims, block, stride, nullptr, nullptr, nullptr, &scr);
  if (rc) return rc;
  if (!bytes) return fail(XATTN_ERR_ARG, "bytes is NULL");
  XattnShape s;
  check_dims(dims, &s);
  *bytes = scr + score_scratch_bytes(s, stride);
  return ok();
}

int xattn_forward(const void* q, const void* k, const void* v, const xattn_dims* dims, int block,
                  int stride, float tau, void* o, float* lse, void* workspace,
                  size_t workspace_bytes, void* stream) {
  XattnShape s;
  int rc;
  if ((rc = check_dims(dims, &s)) || (rc = check_block(block)) || (rc = check_stride(stride)) ||
      (rc = check_tau(tau)))
    return rc;
  if (!q || !k || !v || !o) return fail(XATTN_ERR_ARG, "q, k, v and o must be non-NULL");
  size_t o_sc, o_idx, o_cnt, o_scr, need;
  xattn_forward_layout(dims, block, stride, &o_sc, &o_idx, &o_cnt, &o_scr);
  need = o_scr + score_scratch_bytes(s, stride);
  if (!workspace || workspace_bytes < need)
    return fail(XATTN_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                workspace ? workspace_bytes : (size_t)0);
  char* ws = (char*)workspace;
  float* sc = (float*)(ws + o_sc);
  int32_t* idx = (int32_t*)(ws + o_idx);
  int32_t* cnt = (int32_t*)(ws + o_cnt);
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = launch_score(q, k, s, stride, nullptr, sc, ws + o_scr, st);
  if (e == hipSuccess) e = launch_select(sc, s, uniform_threshold(s, tau), idx, cnt, st);
  if (e == hipSuccess) e = launch_attn(q, k, v, s, idx, cnt, false, o, lse, st);
  return hip_status(e, "xattn_forward launch");
}

int xattn_forward_noalloc(const void* q, const void* k, const void* v, const xattn_dims* dims,
                          int block, int stride, float tau, void* o, float* lse, void* stream) {
  static_assert(kNoallocScratchBytes == XATTN_NOALLOC_SCRATCH_BYTES, "header and library agree");
  XattnShape s;
  int rc;
  if ((rc = check_dims(dims, &s)) || (rc = check_block(block)) || (rc = check_stride(stride)) ||
      (rc = check_tau(tau)))
    return rc;
  if (!q || !k || !v || !o) return fail(XATTN_ERR_ARG, "q, k, v and o must be non-NULL");
  size_t need = 0;
  if ((rc = xattn_forward_workspace_size(dims, block, stride, &need))) return rc;
  if (need > kNoallocScratchBytes)
    return fail(XATTN_ERR_UNSUPPORTED,
                "this problem needs %zu bytes of scratch; xattn_forward_noalloc holds %zu "
                "(use xattn_forward with a caller workspace)",
                need, kNoallocScratchBytes);
  void* ws = nullptr;
  if (hipError_t e = noalloc_scratch(&ws); e != hipSuccess)
    return hip_status(e, "xattn_forward_noalloc: address of the static scratch");
  return xattn_forward(q, k, v, dims, block, stride, tau, o, lse, ws, kNoallocScratchBytes,
                       stream);
}

int xattn_forward_scheduled(const void* q, const void* k, const void* v, const xattn_dims* dims,
                            int block, int stride, float tau, int step, int warmup_steps,
                            void* o, float* lse, void* workspace, size_t workspace_bytes,
                            void* stream) {
  if (step < 0) return fail(XATTN_ERR_ARG, "step must be >= 0 (got %d)", step);
  if (warmup_steps < 0)
    return fail(XATTN_ERR_ARG, "warmup_steps must be >= 0 (got %d)", warmup_steps);
  if (step < warmup_steps) {
    XattnShape s;
    int rc;
    if ((rc = check_dims(dims, &s)) || (rc = check_block(block)) || (rc = check_stride(stride)) ||
        (rc = check_tau(tau)))
      return rc;
    return xattn_dense_attn(q, k, v, dims, o, lse, stream);
  }
  return xattn_forward(q, k, v, dims, block, stride, tau, o, lse, workspace, workspace_bytes,
                       stream);
}

int xattn_head_error_workspace_size(const xattn_dims* dims, size_t* bytes) {
  XattnShape s;
  int rc;
  if ((rc = check_dims(dims, &s))) return rc;
  if (!bytes) return fail(XATTN_ERR_ARG, "bytes is NULL");
  *bytes = head_error_scratch_bytes(s);
  return ok();
}

static int head_error_common(const void* o, const void* o_ref, const xattn_dims* dims,
                             double* err, void* workspace, size_t workspace_bytes,
                             bool mean_over_batch, void* stream) {
  XattnShape s;
  int rc;
  if ((rc = check_dims(dims, &s))) return rc;
  if (s.HQ() > 65535) return fail(XATTN_ERR_UNSUPPORTED, "more than 65535 heads");
  if (!o || !o_ref || !err) return fail(XATTN_ERR_ARG, "o, o_ref and err must be non-NULL");
  const size_t need = head_error_scratch_bytes(s);
  if (!workspace || workspace_bytes < need)
    return fail(XATTN_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                workspace ? workspace_bytes : (size_t)0);
  return hip_status(launch_head_error(o, o_ref, s, err, workspace, mean_over_batch,
                                      (hipStream_t)stream),
                    "xattn_head_error launch");
}

int xattn_head_error(const void* o, const void* o_ref, const xattn_dims* dims, double* err,
                     void* workspace, size_t workspace_bytes, void* stream) {
  return head_error_common(o, o_ref, dims, err, workspace, workspace_bytes, false, stream);
}

int xattn_head_error_mean(const void* o, const void* o_ref, const xattn_dims* dims,
                          double* err, void* workspace, size_t workspace_bytes, void* stream) {
  return head_error_common(o, o_ref, dims, err, workspace, workspace_bytes, true, stream);
}

const char* xattn_strerror(int status) {
  switch (status) {
    case XATTN_OK: return "ok";
    case XATTN_ERR_ARG: return "invalid argument";
    case XATTN_ERR_UNSUPPORTED: return "unsupported configuration";
    case XATTN_ERR_WORKSPACE: return "workspace missing or too small";
    case XATTN_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* xattn_last_error(void) { return g_err; }

int xattn_version(void) { return 10100; }

}  // extern "C"
