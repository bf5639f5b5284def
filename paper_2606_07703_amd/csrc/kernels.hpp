// Internal launch interface between the C ABI (api.cpp) and the kernels.
// Every launcher assumes its problem has been validated by the host layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sparse_prefill.h"

namespace sp {

// A validated problem with defaults resolved.
struct Prob {
  int S, Hq, Hkv, G, d, di, k, b, R, W, agg, relu, dtype;
  int ha;        // head axis: 0 one support shared by all heads, 1 one per KV group
  int qo;        // position of the first query row (a chunk [qo, S) of the sequence)
  int nq;        // query rows, S - qo; R counts the chunk's selection blocks
  float scale;   // attention logit scale
  float iscale;  // indexer score scale
  // elements between the support tables of consecutive KV groups
  size_t idx_group_stride() const { return ha ? (size_t)R * k : 0; }
};

// K/V storage of the sparse attention kernels: contiguous rows (table ==
// nullptr) or a paged cache where token s lives in row
// table[s / page_size] * page_size + s % page_size of num_pages * page_size.
struct KvPages {
  const int32_t *table = nullptr;
  int page_size = 0;
  int num_pages = 0;
  __device__ __forceinline__ int row(int s) const {
    if (!table) return s;
    const int pg = table[s / page_size];
    return (pg >= 0 && pg < num_pages) ? pg * page_size + s % page_size : -1;
  }
};

// Dense (idx == nullptr) or sparse (idx != nullptr) attention, one wave per
// (query, head chunk). o and/or lse may be null.
hipError_t launch_attn_rowwise(const Prob &p, const void *q, const void *k, const void *v,
                               const int32_t *idx, void *o, float *lse, hipStream_t st,
                               KvPages pages = KvPages());

// bf16 MFMA sparse attention for selection blocks of b >= 16 queries: each
// gathered K/V row is shared by the b*G query rows of a KV head.
bool sparse_query_mfma_supported(const Prob &p);
hipError_t launch_sparse_query_mfma(const Prob &p, const void *q, const void *k, const void *v,
                                    const int32_t *idx, void *o, hipStream_t st,
                                    KvPages pages = KvPages());
// paged: K/V read through a page table (a smaller support fits LDS at d = 256)
bool sparse_block_mfma_supported(const Prob &p, bool paged);
hipError_t launch_sparse_block_mfma(const Prob &p, const void *q, const void *k, const void *v,
                                    const int32_t *idx, void *o, hipStream_t st,
                                    KvPages pages = KvPages());

// bf16 MFMA causal flash attention; o and/or lse (o == nullptr: normalisers only).
bool dense_mfma_supported(const Prob &p);
hipError_t launch_dense_mfma(const Prob &p, const void *q, const void *k, const void *v,
                             void *o, float *lse, hipStream_t st);

// Head-averaged mass with block aggregation.
hipError_t launch_mass_rowwise(const Prob &p, const void *q, const void *k, const float *lse,
                               float *mass, hipStream_t st);
bool mass_mfma_supported(const Prob &p);
hipError_t launch_mass_mfma(const Prob &p, const void *q, const void *k, const float *lse,
                            float *mass, hipStream_t st);

// Indexer scores with block aggregation.
hipError_t launch_indexer_rowwise(const Prob &p, const void *qi, const void *ki, float *scores,
                                  hipStream_t st);

// bf16 MFMA indexer scores: b = 1 stores every causal score, b in
// {16, 32, 64, 128} reduces over each selection block in the epilogue.
bool indexer_mfma_supported(const Prob &p);
hipError_t launch_indexer_mfma(const Prob &p, const void *qi, const void *ki, float *scores,
                               hipStream_t st);

// Row-wise top-k selection.
hipError_t launch_indexer_project(int S, int di, int dm, int pos0, float theta, float eps,
                                  const void *x, const void *wq, const void *wk,
                                  const float *gamma, const float *beta, void *qo, void *ko,
                                  hipStream_t st);
bool indexer_topk_supported(const Prob &p);
size_t indexer_topk_workspace(const Prob &p);
hipError_t launch_indexer_topk(const Prob &p, const void *qi, const void *ki, int32_t *idx,
                               void *ws, hipStream_t st);
// The same with its scratch in a static device array of this many bytes (per
// GPU); problems whose workspace exceeds it are refused by the API.
constexpr size_t kIndexerTopkStaticBytes = size_t(64) << 20;
hipError_t launch_indexer_topk_static(const Prob &p, const void *qi, const void *ki,
                                      int32_t *idx, hipStream_t st);
hipError_t launch_kl_loss(int S, int n, const int32_t *rows, const float *P, const float *z,
                          float *kl, float *loss, float *grad, hipStream_t st);
hipError_t launch_topk(const Prob &p, const float *scores, int32_t *idx, hipStream_t st);

}  // namespace sp
