// Drives every C ABI entry point through validation and dispatch, on the
// host, against the stand-ins of abi_stubs.cpp. Built with AddressSanitizer
// and UBSan: any invalid access or undefined operation in the host layer
// aborts the run. Prints "abi ok" and exits 0 when every check holds.
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "kernels.hpp"
#include "sparse_prefill.h"

namespace stub {
extern int have_device;
extern const char *arch;
extern const char *last;
extern sp::Prob prob;
extern int calls;
}  // namespace stub

static int failures = 0;
#define CHECK(cond)                                                  \
  do {                                                               \
    if (!(cond)) {                                                   \
      fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                    \
    }                                                                \
  } while (0)

// Distinct 16-byte aligned addresses that are never dereferenced.
static void *addr(int i) { return (void *)(uintptr_t)(0x100000 * (i + 1)); }

static sp_problem base() {
  sp_problem p;
  memset(&p, 0, sizeof(p));
  p.seq_len = 300;
  p.num_q_heads = 8;
  p.num_kv_heads = 2;
  p.head_dim = 128;
  p.index_dim = 64;
  p.topk = 32;
  p.block_q = 16;
  p.causal = 1;
  p.dtype = SP_DTYPE_BF16;
  return p;
}

static int dense(const sp_problem *p) {
  return sp_dense_attn(p, addr(0), addr(1), addr(2), addr(3), (float *)addr(4), nullptr);
}
static int sparse(const sp_problem *p) {
  return sp_sparse_gqa_attn(p, addr(0), addr(1), addr(2), (const int32_t *)addr(3), addr(4),
                            nullptr);
}
static int indexer(const sp_problem *p) {
  return sp_indexer_scores(p, addr(0), addr(1), (float *)addr(2), nullptr);
}
static int topk(const sp_problem *p) {
  return sp_topk_select(p, (const float *)addr(0), (int32_t *)addr(1), nullptr, 0, nullptr);
}
static int mass(const sp_problem *p) {
  return sp_oracle_support(p, addr(0), addr(1), (const float *)addr(2), (float *)addr(3),
                           nullptr);
}

int main() {
  // every status has a message; unknown codes are named as such
  for (int s = 0; s >= -8; --s) CHECK(strcmp(sp_status_string(s), "unknown status") != 0);
  CHECK(strcmp(sp_status_string(5), "unknown status") == 0);
  CHECK(sp_version() == SP_VERSION);

  // NULL problem
  CHECK(dense(nullptr) == SP_ERR_NULL);
  CHECK(sparse(nullptr) == SP_ERR_NULL);
  CHECK(indexer(nullptr) == SP_ERR_NULL);
  CHECK(topk(nullptr) == SP_ERR_NULL);
  CHECK(mass(nullptr) == SP_ERR_NULL);
  size_t ws = 0;
  CHECK(sp_workspace_bytes(nullptr, SP_OP_TOPK, &ws) == SP_ERR_NULL);

  // valid calls reach a launcher with defaults resolved
  sp_problem p = base();
  stub::calls = 0;
  CHECK(dense(&p) == SP_OK && strcmp(stub::last, "dense_mfma") == 0);
  CHECK(fabsf(stub::prob.scale - 1.f / sqrtf(128.f)) < 1e-7f);
  CHECK(stub::prob.G == 4 && stub::prob.R == (300 + 15) / 16 && stub::prob.nq == 300);
  CHECK(sparse(&p) == SP_OK && strcmp(stub::last, "sparse_block_mfma") == 0);
  CHECK(indexer(&p) == SP_OK && strcmp(stub::last, "indexer_mfma") == 0);
  CHECK(fabsf(stub::prob.iscale - 1.f / sqrtf(64.f)) < 1e-7f);
  CHECK(topk(&p) == SP_OK && strcmp(stub::last, "topk") == 0);
  CHECK(mass(&p) == SP_OK && strcmp(stub::last, "mass_mfma") == 0);
  CHECK(stub::calls == 5);

  // chunked call: R counts the chunk's blocks
  p = base();
  p.q_offset = 64;
  CHECK(sparse(&p) == SP_OK && stub::prob.qo == 64 && stub::prob.nq == 236 &&
        stub::prob.R == (236 + 15) / 16);
  p.q_offset = 60;   // not on a block boundary
  CHECK(sparse(&p) == SP_ERR_SHAPE);
  p.q_offset = 300;
  CHECK(sparse(&p) == SP_ERR_SHAPE);

  // per-query selection takes the per-query kernel; fp32 the row-wise one
  p = base();
  p.block_q = 1;
  CHECK(sparse(&p) == SP_OK && strcmp(stub::last, "sparse_query_mfma") == 0);
  p.dtype = SP_DTYPE_F32;
  CHECK(sparse(&p) == SP_OK && strcmp(stub::last, "attn_rowwise_sparse") == 0);
  CHECK(dense(&p) == SP_OK && strcmp(stub::last, "attn_rowwise_dense") == 0);

  // shape and scale errors
  p = base();
  p.num_q_heads = 7;
  CHECK(dense(&p) == SP_ERR_SHAPE);
  p = base();
  p.attn_scale = -0.5f;
  CHECK(dense(&p) == SP_ERR_SHAPE && sparse(&p) == SP_ERR_SHAPE && mass(&p) == SP_ERR_SHAPE);
  p.attn_scale = NAN;
  CHECK(dense(&p) == SP_ERR_SHAPE);
  p.attn_scale = INFINITY;
  CHECK(dense(&p) == SP_ERR_SHAPE);
  p = base();
  p.attn_scale = 0.25f;
  CHECK(dense(&p) == SP_OK && stub::prob.scale == 0.25f);
  p = base();
  p.topk = 0;
  CHECK(sparse(&p) == SP_ERR_SHAPE && topk(&p) == SP_ERR_SHAPE);
  p = base();
  p.local_window = 33;
  CHECK(topk(&p) == SP_ERR_SHAPE);
  p = base();
  p.causal = 0;
  CHECK(dense(&p) == SP_ERR_UNSUPPORTED);
  p = base();
  p.head_dim = 96;
  CHECK(dense(&p) == SP_ERR_UNSUPPORTED);
  p = base();
  p.agg = 2;
  CHECK(indexer(&p) == SP_ERR_SHAPE);
  p = base();
  p.relu = 2;
  CHECK(indexer(&p) == SP_ERR_SHAPE);
  // sizes at the int32 limits: K/V of 4 GiB or more are refused, not wrapped
  p = base();
  p.seq_len = 2147483647;
  p.num_kv_heads = 8;
  p.num_q_heads = 8;
  CHECK(dense(&p) == SP_ERR_UNSUPPORTED);
  p = base();
  p.seq_len = 2147483647;
  p.block_q = 2147483647;
  p.topk = 2147483647;
  CHECK(topk(&p) == SP_OK && stub::prob.R == 1);

  // alignment and NULL outputs
  p = base();
  CHECK(sp_dense_attn(&p, (char *)addr(0) + 8, addr(1), addr(2), addr(3), nullptr, nullptr) ==
        SP_ERR_ALIGN);
  CHECK(sp_dense_attn(&p, addr(0), addr(1), addr(2), nullptr, nullptr, nullptr) == SP_ERR_NULL);

  // workspace of the fused scoring + top-k
  p = base();
  p.block_q = 1;
  CHECK(sp_workspace_bytes(&p, SP_OP_INDEXER_TOPK, &ws) == SP_OK && ws == 300u * 1024u);
  CHECK(sp_indexer_topk(&p, addr(0), addr(1), (int32_t *)addr(2), addr(3), ws - 16, nullptr) ==
        SP_ERR_WORKSPACE);
  CHECK(sp_indexer_topk(&p, addr(0), addr(1), (int32_t *)addr(2), addr(3), ws, nullptr) ==
        SP_OK);
  CHECK(sp_workspace_bytes(&p, 99, &ws) == SP_ERR_SHAPE);
  // the allocation-free variant: same validation, its scratch bounded by the
  // static array (the stand-in workspace is S * 1024 bytes)
  CHECK(sp_indexer_topk_noalloc(&p, addr(0), addr(1), (int32_t *)addr(2), nullptr) == SP_OK &&
        strcmp(stub::last, "indexer_topk_static") == 0);
  p.seq_len = 65535;   // 64 MiB of stand-in workspace: exactly at the bound
  CHECK(sp_indexer_topk_noalloc(&p, addr(0), addr(1), (int32_t *)addr(2), nullptr) == SP_OK);
  p.seq_len = 65536;   // past the fused kernel's limit
  CHECK(sp_indexer_topk_noalloc(&p, addr(0), addr(1), (int32_t *)addr(2), nullptr) ==
        SP_ERR_UNSUPPORTED);
  p = base();
  p.block_q = 1;
  CHECK(sp_indexer_topk_noalloc(&p, nullptr, addr(1), (int32_t *)addr(2), nullptr) ==
        SP_ERR_NULL);
  p.block_q = 4;
  CHECK(sp_indexer_topk_noalloc(&p, addr(0), addr(1), (int32_t *)addr(2), nullptr) ==
        SP_ERR_UNSUPPORTED);

  // KL and the front end
  p = base();
  CHECK(sp_kl_loss(&p, (const int32_t *)addr(0), 0, nullptr, nullptr, nullptr, nullptr, nullptr,
                   nullptr) == SP_OK);
  CHECK(sp_kl_loss(&p, (const int32_t *)addr(0), 4, (const float *)addr(1),
                   (const float *)addr(2), nullptr, (float *)addr(3), nullptr,
                   nullptr) == SP_ERR_NULL);
  CHECK(sp_indexer_project(&p, 4096, 0, 10000.f, 1e-6f, addr(0), addr(1), addr(2),
                           (const float *)addr(3), (const float *)addr(4), addr(5), addr(6),
                           nullptr) == SP_OK);
  CHECK(sp_indexer_project(&p, 4096, 2147483647, 10000.f, 1e-6f, addr(0), addr(1), addr(2),
                           (const float *)addr(3), (const float *)addr(4), addr(5), addr(6),
                           nullptr) == SP_ERR_SHAPE);

  // paged K/V
  p = base();
  CHECK(sp_sparse_gqa_attn_paged(&p, addr(0), addr(1), addr(2), (const int32_t *)addr(3), 64, 8,
                                 (const int32_t *)addr(4), addr(5), nullptr) == SP_OK);
  CHECK(sp_sparse_gqa_attn_paged(&p, addr(0), addr(1), addr(2), (const int32_t *)addr(3), 0, 8,
                                 (const int32_t *)addr(4), addr(5), nullptr) == SP_ERR_SHAPE);

  // device checks come after validation
  p = base();
  stub::have_device = 0;
  CHECK(dense(&p) == SP_ERR_NO_DEVICE);
  p.num_q_heads = 7;
  CHECK(dense(&p) == SP_ERR_SHAPE);

  if (failures) {
    fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  printf("abi ok\n");
  return 0;
}
