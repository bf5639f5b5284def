// Host-only stand-ins for the HIP runtime calls and the kernel launchers
// that the C ABI layer (api.cpp) reaches after validation. Linked with
// api.cpp into a sanitizer build, they let every entry point run to its
// dispatch without a GPU: each launcher records its name and the resolved
// problem instead of launching.
#include <hip/hip_runtime_api.h>
#include <string.h>

#include "kernels.hpp"

namespace stub {
int have_device = 1;              // hipGetDevice succeeds
const char *arch = "gfx950:sramecc+:xnack-";
const char *last = "";            // name of the last launcher called
sp::Prob prob;                    // the problem it received
int calls = 0;
}  // namespace stub

extern "C" {
hipError_t hipGetDevice(int *dev) {
  if (!stub::have_device) return hipErrorNoDevice;
  *dev = 0;
  return hipSuccess;
}
hipError_t hipGetDevicePropertiesR0600(hipDeviceProp_tR0600 *prop, int) {
  memset(prop, 0, sizeof(*prop));
  strncpy(prop->gcnArchName, stub::arch, sizeof(prop->gcnArchName) - 1);
  return hipSuccess;
}
hipError_t hipGetLastError(void) { return hipSuccess; }
}

namespace sp {
namespace {
hipError_t record(const char *name, const Prob &p);
}  // namespace
}  // namespace sp

namespace sp {
namespace {
hipError_t record(const char *name, const Prob &p) {
  stub::last = name;
  stub::prob = p;
  ++stub::calls;
  return hipSuccess;
}
}  // namespace

hipError_t launch_attn_rowwise(const Prob &p, const void *, const void *, const void *,
                               const int32_t *idx, void *, float *, hipStream_t, KvPages) {
  return record(idx ? "attn_rowwise_sparse" : "attn_rowwise_dense", p);
}
bool sparse_query_mfma_supported(const Prob &p) { return p.dtype == SP_DTYPE_BF16; }
hipError_t launch_sparse_query_mfma(const Prob &p, const void *, const void *, const void *,
                                    const int32_t *, void *, hipStream_t, KvPages) {
  return record("sparse_query_mfma", p);
}
bool sparse_block_mfma_supported(const Prob &p, bool) {
  return p.dtype == SP_DTYPE_BF16 && p.b >= 16;
}
hipError_t launch_sparse_block_mfma(const Prob &p, const void *, const void *, const void *,
                                    const int32_t *, void *, hipStream_t, KvPages) {
  return record("sparse_block_mfma", p);
}
bool dense_mfma_supported(const Prob &p) { return p.dtype == SP_DTYPE_BF16; }
hipError_t launch_dense_mfma(const Prob &p, const void *, const void *, const void *, void *,
                             float *, hipStream_t) {
  return record("dense_mfma", p);
}
hipError_t launch_mass_rowwise(const Prob &p, const void *, const void *, const float *,
                               float *, hipStream_t) {
  return record("mass_rowwise", p);
}
bool mass_mfma_supported(const Prob &p) { return p.dtype == SP_DTYPE_BF16; }
hipError_t launch_mass_mfma(const Prob &p, const void *, const void *, const float *, float *,
                            hipStream_t) {
  return record("mass_mfma", p);
}
hipError_t launch_indexer_rowwise(const Prob &p, const void *, const void *, float *,
                                  hipStream_t) {
  return record("indexer_rowwise", p);
}
bool indexer_mfma_supported(const Prob &p) { return p.dtype == SP_DTYPE_BF16; }
hipError_t launch_indexer_mfma(const Prob &p, const void *, const void *, float *,
                               hipStream_t) {
  return record("indexer_mfma", p);
}
hipError_t launch_indexer_project(int S, int di, int, int, float, float, const void *,
                                  const void *, const void *, const float *, const float *,
                                  void *, void *, hipStream_t) {
  Prob p{};
  p.S = S;
  p.di = di;
  return record("indexer_project", p);
}
bool indexer_topk_supported(const Prob &p) { return p.S <= 65535; }
size_t indexer_topk_workspace(const Prob &p) { return (size_t)p.S * 1024; }
hipError_t launch_indexer_topk(const Prob &p, const void *, const void *, int32_t *, void *,
                               hipStream_t) {
  return record("indexer_topk", p);
}
hipError_t launch_kl_loss(int S, int, const int32_t *, const float *, const float *, float *,
                          float *, float *, hipStream_t) {
  Prob p{};
  p.S = S;
  return record("kl_loss", p);
}
hipError_t launch_topk(const Prob &p, const float *, int32_t *, hipStream_t) {
  return record("topk", p);
}
}  // namespace sp

namespace sp {
hipError_t launch_indexer_topk_static(const Prob &p, const void *, const void *, int32_t *,
                                      hipStream_t) {
  return record("indexer_topk_static", p);
}
}  // namespace sp
