// The C ABI: argument validation (host only, before any HIP call), device
// checks, and dispatch to the gfx950 kernels. Nothing here allocates device
// memory or synchronises.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <atomic>

#include "kernels.hpp"
#include "sparse_prefill.h"

namespace sp {
namespace {

constexpr int kMaxDevices = 64;
// 0 = unknown, 1 = gfx950, 2 = other architecture.
std::atomic<int> g_arch[kMaxDevices];

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Shape fields every operation uses.
int check_common(const sp_problem *p) {
  if (!p) return SP_ERR_NULL;
  if (p->seq_len < 1 || p->num_q_heads < 1 || p->num_kv_heads < 1) return SP_ERR_SHAPE;
  if (p->q_offset < 0 || p->q_offset >= p->seq_len) return SP_ERR_SHAPE;
  if (p->num_q_heads % p->num_kv_heads != 0) return SP_ERR_SHAPE;
  if (p->causal != 1) return SP_ERR_UNSUPPORTED;
  if (p->dtype != SP_DTYPE_F32 && p->dtype != SP_DTYPE_BF16) return SP_ERR_UNSUPPORTED;
  if (!isfinite(p->attn_scale) || !isfinite(p->index_scale)) return SP_ERR_SHAPE;
  // The attention kernels take row maxima of raw scores and scale them
  // afterwards, which needs scale >= 0 (the paper's 1/sqrt(d) is positive).
  if (p->attn_scale < 0.f) return SP_ERR_SHAPE;
  return SP_OK;
}

int check_heads(const sp_problem *p) {
  if (p->head_dim != 64 && p->head_dim != 128 && p->head_dim != 256) return SP_ERR_UNSUPPORTED;
  // K and V rows are addressed with 32-bit byte offsets.
  const int64_t elt = p->dtype == SP_DTYPE_BF16 ? 2 : 4;
  if ((int64_t)p->seq_len * p->num_kv_heads * p->head_dim * elt >= (int64_t(1) << 32))
    return SP_ERR_UNSUPPORTED;
  // The row-wise oracle kernel stages one query's heads in 64 KiB of LDS.
  if ((int64_t)p->num_q_heads * (p->head_dim + 1) * 4 > 65536) return SP_ERR_UNSUPPORTED;
  return SP_OK;
}

int check_selection(const sp_problem *p) {
  if (p->block_q < 1) return SP_ERR_SHAPE;
  if (p->head_axis != 0 && p->head_axis != 1) return SP_ERR_SHAPE;
  // a chunk starts on a selection-block boundary
  if (p->q_offset % p->block_q != 0) return SP_ERR_SHAPE;
  if (p->topk < 1) return SP_ERR_SHAPE;
  if (p->local_window < 0 || p->local_window > p->topk) return SP_ERR_SHAPE;
  return SP_OK;
}

int check_agg(const sp_problem *p) {
  if (p->agg != SP_AGG_MAX && p->agg != SP_AGG_SUM) return SP_ERR_SHAPE;
  return SP_OK;
}

Prob resolve(const sp_problem *p) {
  Prob r;
  r.S = p->seq_len;
  r.Hq = p->num_q_heads;
  r.Hkv = p->num_kv_heads;
  r.G = r.Hq / r.Hkv;
  r.d = p->head_dim;
  r.di = p->index_dim;
  r.k = p->topk;
  r.qo = p->q_offset;
  r.nq = r.S - r.qo;
  // a block longer than the call's rows is one block of all of them (same
  // result, and no kernel forms b * G or t0 + b beyond int range)
  r.b = p->block_q < 1 ? 1 : p->block_q < r.nq ? p->block_q : r.nq;
  r.R = r.nq / r.b + (r.nq % r.b != 0);
  r.W = p->local_window;
  r.agg = p->agg;
  r.relu = p->relu;
  r.dtype = p->dtype;
  r.ha = p->head_axis;
  r.scale = p->attn_scale != 0.f ? p->attn_scale : 1.f / sqrtf((float)(r.d > 0 ? r.d : 1));
  r.iscale = p->index_scale != 0.f ? p->index_scale : 1.f / sqrtf((float)(r.di > 0 ? r.di : 1));
  return r;
}

// Device and architecture check, after validation.
int check_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
    (void)hipGetLastError();
    return SP_ERR_NO_DEVICE;
  }
  if (dev >= kMaxDevices) return SP_ERR_NO_DEVICE;
  int a = g_arch[dev].load(std::memory_order_relaxed);
  if (a == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) {
      (void)hipGetLastError();
      return SP_ERR_NO_DEVICE;
    }
    a = strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 2;
    g_arch[dev].store(a, std::memory_order_relaxed);
  }
  return a == 1 ? SP_OK : SP_ERR_ARCH;
}

int launched(hipError_t e) { return e == hipSuccess ? SP_OK : SP_ERR_HIP; }

#define SP_TRY(expr)          \
  do {                        \
    const int _rc = (expr);   \
    if (_rc != SP_OK) return _rc; \
  } while (0)

}  // namespace
}  // namespace sp

using namespace sp;

extern "C" {

int sp_dense_attn(const sp_problem *p, const void *q, const void *k, const void *v, void *o,
                  float *lse, hipStream_t stream) {
  SP_TRY(check_common(p));
  SP_TRY(check_heads(p));
  if (!q || !k || !v || (!o && !lse)) return SP_ERR_NULL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(lse))
    return SP_ERR_ALIGN;
  SP_TRY(check_device());
  const Prob r = resolve(p);
  if (r.qo == 0 && dense_mfma_supported(r))
    return launched(launch_dense_mfma(r, q, k, v, o, lse, stream));
  return launched(launch_attn_rowwise(r, q, k, v, nullptr, o, lse, stream));
}

int sp_oracle_support(const sp_problem *p, const void *q, const void *k, const float *lse,
                      float *mass, hipStream_t stream) {
  SP_TRY(check_common(p));
  SP_TRY(check_heads(p));
  SP_TRY(check_selection(p));
  SP_TRY(check_agg(p));
  if (p->q_offset != 0) return SP_ERR_UNSUPPORTED;   // the oracle runs on whole sequences
  if (!q || !k || !lse || !mass) return SP_ERR_NULL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(lse) || !aligned16(mass)) return SP_ERR_ALIGN;
  SP_TRY(check_device());
  const Prob r = resolve(p);
  if (!r.ha && mass_mfma_supported(r))
    return launched(launch_mass_mfma(r, q, k, lse, mass, stream));
  return launched(launch_mass_rowwise(r, q, k, lse, mass, stream));
}

int sp_indexer_scores(const sp_problem *p, const void *q_idx, const void *k_idx, float *scores,
                      hipStream_t stream) {
  SP_TRY(check_common(p));
  SP_TRY(check_selection(p));
  if (p->head_axis != 0) return SP_ERR_UNSUPPORTED;   // the indexer is head-collapsed
  SP_TRY(check_agg(p));
  if (p->index_dim != 64 && p->index_dim != 128 && p->index_dim != 256)
    return SP_ERR_UNSUPPORTED;
  if (p->relu != 0 && p->relu != 1) return SP_ERR_SHAPE;
  if (!q_idx || !k_idx || !scores) return SP_ERR_NULL;
  if (!aligned16(q_idx) || !aligned16(k_idx) || !aligned16(scores)) return SP_ERR_ALIGN;
  SP_TRY(check_device());
  const Prob r = resolve(p);
  if (indexer_mfma_supported(r))
    return launched(launch_indexer_mfma(r, q_idx, k_idx, scores, stream));
  return launched(launch_indexer_rowwise(r, q_idx, k_idx, scores, stream));
}

int sp_topk_select(const sp_problem *p, const float *scores, int32_t *idx, void *workspace,
                   size_t workspace_bytes, hipStream_t stream) {
  SP_TRY(check_common(p));
  SP_TRY(check_selection(p));
  if (!scores || !idx) return SP_ERR_NULL;
  if (!aligned16(scores) || !aligned16(idx) || !aligned16(workspace)) return SP_ERR_ALIGN;
  size_t need = 0;
  SP_TRY(sp_workspace_bytes(p, SP_OP_TOPK, &need));
  if (need > 0 && (!workspace || workspace_bytes < need)) return SP_ERR_WORKSPACE;
  SP_TRY(check_device());
  const Prob r = resolve(p);
  return launched(launch_topk(r, scores, idx, stream));
}

int sp_sparse_gqa_attn(const sp_problem *p, const void *q, const void *k, const void *v,
                       const int32_t *idx, void *o, hipStream_t stream) {
  SP_TRY(check_common(p));
  SP_TRY(check_heads(p));
  SP_TRY(check_selection(p));
  if (!q || !k || !v || !idx || !o) return SP_ERR_NULL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(idx) || !aligned16(o))
    return SP_ERR_ALIGN;
  SP_TRY(check_device());
  const Prob r = resolve(p);
  if (sparse_block_mfma_supported(r, false))
    return launched(launch_sparse_block_mfma(r, q, k, v, idx, o, stream));
  if (sparse_query_mfma_supported(r))
    return launched(launch_sparse_query_mfma(r, q, k, v, idx, o, stream));
  return launched(launch_attn_rowwise(r, q, k, v, idx, o, nullptr, stream));
}

int sp_indexer_topk(const sp_problem *p, const void *q_idx, const void *k_idx, int32_t *idx,
                    void *workspace, size_t workspace_bytes, hipStream_t stream) {
  SP_TRY(check_common(p));
  SP_TRY(check_selection(p));
  if (p->head_axis != 0) return SP_ERR_UNSUPPORTED;   // the indexer is head-collapsed
  if (p->index_dim != 64 && p->index_dim != 128 && p->index_dim != 256)
    return SP_ERR_UNSUPPORTED;
  if (p->relu != 0 && p->relu != 1) return SP_ERR_SHAPE;
  if (p->block_q != 1) return SP_ERR_UNSUPPORTED;   // the block form aggregates in-kernel
  if (p->q_offset != 0) return SP_ERR_UNSUPPORTED;
  if (!q_idx || !k_idx || !idx) return SP_ERR_NULL;
  if (!aligned16(q_idx) || !aligned16(k_idx) || !aligned16(idx) || !aligned16(workspace))
    return SP_ERR_ALIGN;
  const Prob r = resolve(p);
  if (!indexer_topk_supported(r)) return SP_ERR_UNSUPPORTED;
  size_t need = 0;
  SP_TRY(sp_workspace_bytes(p, SP_OP_INDEXER_TOPK, &need));
  if (!workspace || workspace_bytes < need) return SP_ERR_WORKSPACE;
  SP_TRY(check_device());
  return launched(launch_indexer_topk(r, q_idx, k_idx, idx, workspace, stream));
}

int sp_indexer_topk_noalloc(const sp_problem *p, const void *q_idx, const void *k_idx,
                            int32_t *idx, hipStream_t stream) {
  SP_TRY(check_common(p));
  SP_TRY(check_selection(p));
  if (p->head_axis != 0) return SP_ERR_UNSUPPORTED;
  if (p->index_dim != 64 && p->index_dim != 128 && p->index_dim != 256)
    return SP_ERR_UNSUPPORTED;
  if (p->relu != 0 && p->relu != 1) return SP_ERR_SHAPE;
  if (p->block_q != 1) return SP_ERR_UNSUPPORTED;
  if (p->q_offset != 0) return SP_ERR_UNSUPPORTED;
  if (!q_idx || !k_idx || !idx) return SP_ERR_NULL;
  if (!aligned16(q_idx) || !aligned16(k_idx) || !aligned16(idx)) return SP_ERR_ALIGN;
  const Prob r = resolve(p);
  if (!indexer_topk_supported(r)) return SP_ERR_UNSUPPORTED;
  // the scratch this call needs must fit the library's static array
  if (indexer_topk_workspace(r) > kIndexerTopkStaticBytes) return SP_ERR_WORKSPACE;
  SP_TRY(check_device());
  return launched(launch_indexer_topk_static(r, q_idx, k_idx, idx, stream));
}

int sp_indexer_project(const sp_problem *p, int32_t d_model, int32_t pos0, float rope_theta,
                       float ln_eps, const void *x, const void *w_q, const void *w_k,
                       const float *gamma, const float *beta, void *q_idx, void *k_idx,
                       hipStream_t stream) {
  if (!p) return SP_ERR_NULL;
  if (p->seq_len < 1 || d_model < 1 || pos0 < 0) return SP_ERR_SHAPE;
  if ((int64_t)pos0 + p->seq_len > INT32_MAX) return SP_ERR_SHAPE;
  if (!(rope_theta > 0.f) || !isfinite(rope_theta) || !(ln_eps >= 0.f) || !isfinite(ln_eps))
    return SP_ERR_SHAPE;
  if (p->dtype != SP_DTYPE_BF16) return SP_ERR_UNSUPPORTED;
  if (p->index_dim != 64 && p->index_dim != 128 && p->index_dim != 256) return SP_ERR_UNSUPPORTED;
  if (d_model % 64 != 0) return SP_ERR_UNSUPPORTED;
  if (!x || !w_q || !w_k || !gamma || !beta || !q_idx || !k_idx) return SP_ERR_NULL;
  if (!aligned16(x) || !aligned16(w_q) || !aligned16(w_k) || !aligned16(gamma) ||
      !aligned16(beta) || !aligned16(q_idx) || !aligned16(k_idx))
    return SP_ERR_ALIGN;
  SP_TRY(check_device());
  return launched(launch_indexer_project(p->seq_len, p->index_dim, d_model, pos0, rope_theta,
                                         ln_eps, x, w_q, w_k, gamma, beta, q_idx, k_idx,
                                         stream));
}

int sp_kl_loss(const sp_problem *p, const int32_t *rows, int32_t n_rows, const float *P,
               const float *z, float *kl, float *loss, float *grad_z, hipStream_t stream) {
  if (!p) return SP_ERR_NULL;
  if (p->seq_len < 1 || n_rows < 0) return SP_ERR_SHAPE;
  if (n_rows == 0) return SP_OK;
  if (!rows || !P || !z) return SP_ERR_NULL;
  if (loss && !kl) return SP_ERR_NULL;   // the mean is taken over the per-row values
  if (!aligned16(rows) || !aligned16(P) || !aligned16(z) || !aligned16(kl) ||
      !aligned16(loss) || !aligned16(grad_z))
    return SP_ERR_ALIGN;
  SP_TRY(check_device());
  return launched(launch_kl_loss(p->seq_len, n_rows, rows, P, z, kl, loss, grad_z, stream));
}

int sp_sparse_gqa_attn_paged(const sp_problem *p, const void *q, const void *k_pages,
                             const void *v_pages, const int32_t *page_table, int32_t page_size,
                             int32_t num_pages, const int32_t *idx, void *o,
                             hipStream_t stream) {
  SP_TRY(check_common(p));
  SP_TRY(check_heads(p));
  SP_TRY(check_selection(p));
  if (page_size < 1 || num_pages < 1) return SP_ERR_SHAPE;
  const int64_t elt = p->dtype == SP_DTYPE_BF16 ? 2 : 4;
  if ((int64_t)num_pages * page_size * p->num_kv_heads * p->head_dim * elt >= (int64_t(1) << 32))
    return SP_ERR_UNSUPPORTED;
  if (!q || !k_pages || !v_pages || !page_table || !idx || !o) return SP_ERR_NULL;
  if (!aligned16(q) || !aligned16(k_pages) || !aligned16(v_pages) || !aligned16(page_table) ||
      !aligned16(idx) || !aligned16(o))
    return SP_ERR_ALIGN;
  SP_TRY(check_device());
  const Prob r = resolve(p);
  KvPages pages;
  pages.table = page_table;
  pages.page_size = page_size;
  pages.num_pages = num_pages;
  if (sparse_block_mfma_supported(r, true))
    return launched(launch_sparse_block_mfma(r, q, k_pages, v_pages, idx, o, stream, pages));
  if (sparse_query_mfma_supported(r))
    return launched(launch_sparse_query_mfma(r, q, k_pages, v_pages, idx, o, stream, pages));
  return launched(launch_attn_rowwise(r, q, k_pages, v_pages, idx, o, nullptr, stream, pages));
}

int sp_workspace_bytes(const sp_problem *p, int op, size_t *bytes) {
  if (!p || !bytes) return SP_ERR_NULL;
  if (op < SP_OP_DENSE || op > SP_OP_INDEXER_TOPK) return SP_ERR_SHAPE;
  *bytes = 0;
  if (op == SP_OP_INDEXER_TOPK) {
    SP_TRY(check_common(p));
    *bytes = indexer_topk_workspace(resolve(p));
  }
  return SP_OK;
}

const char *sp_status_string(int status) {
  switch (status) {
    case SP_OK: return "ok";
    case SP_ERR_NULL: return "a required pointer is NULL";
    case SP_ERR_SHAPE: return "inconsistent problem sizes";
    case SP_ERR_UNSUPPORTED: return "unsupported configuration";
    case SP_ERR_WORKSPACE: return "workspace too small";
    case SP_ERR_ALIGN: return "pointer not 16-byte aligned";
    case SP_ERR_NO_DEVICE: return "no usable HIP device";
    case SP_ERR_ARCH: return "device is not gfx950";
    case SP_ERR_HIP: return "HIP launch failed";
    default: return "unknown status";
  }
}

int sp_version(void) { return SP_VERSION; }

}  // extern "C"
