// Host-only stand-ins for the HIP runtime calls and the kernel launchers that sbd_api.cpp
// uses, for the sanitizer build of the C ABI's validation and state machine.  Memory calls
// act on host memory at once (so the sanitizers check every workspace offset the API code
// copies to or fills); launchers do nothing; the device reports no CUs, so no decode path
// that needs them is taken.
#include <cstdlib>
#include <cstring>

#include "hip/hip_runtime.h"
#include "sbd_internal.h"

struct ihipEvent_t {
  int unused;
};

hipError_t hipGetLastError() { return hipSuccess; }
const char* hipGetErrorString(hipError_t e) { return e == hipSuccess ? "no error" : "stub error"; }
hipError_t hipMemcpy(void* dst, const void* src, size_t bytes, hipMemcpyKind) {
  if (bytes && (!dst || !src)) return hipErrorInvalidValue;
  if (bytes) std::memcpy(dst, src, bytes);
  return hipSuccess;
}
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t bytes, hipMemcpyKind kind, hipStream_t) {
  return hipMemcpy(dst, src, bytes, kind);
}
hipError_t hipMemsetAsync(void* dst, int value, size_t bytes, hipStream_t) {
  if (bytes && !dst) return hipErrorInvalidValue;
  if (bytes) std::memset(dst, value, bytes);
  return hipSuccess;
}
hipError_t hipEventCreate(hipEvent_t* e) {
  *e = new ihipEvent_t{0};
  return hipSuccess;
}
hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned) { return hipEventCreate(e); }
hipError_t hipEventDestroy(hipEvent_t e) {
  delete e;
  return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t e, hipStream_t) { return e ? hipSuccess : hipErrorInvalidValue; }
hipError_t hipEventSynchronize(hipEvent_t e) { return e ? hipSuccess : hipErrorInvalidValue; }
hipError_t hipEventElapsedTime(float* ms, hipEvent_t a, hipEvent_t b) {
  if (!a || !b) return hipErrorInvalidValue;
  *ms = 0.f;
  return hipSuccess;
}
hipError_t hipHostMalloc(void** p, size_t bytes, unsigned) {
  *p = std::malloc(bytes ? bytes : 1);
  return *p ? hipSuccess : hipErrorOutOfMemory;
}
hipError_t hipHostFree(void* p) {
  std::free(p);
  return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
hipError_t hipGetDevice(int* dev) {
  *dev = 0;
  return hipSuccess;
}
hipError_t hipDeviceGetAttribute(int* value, hipDeviceAttribute_t, int) {
  *value = 0;
  return hipSuccess;
}

namespace sbd {

GemmPlan gemm_plan(int, int n_tiles, int, int64_t, bool, bool) { return GemmPlan{2, 8, 1, 1, n_tiles / 8}; }
hipError_t launch_gemm(GemmEpi, const GemmArgs&, const Exec&) { return hipSuccess; }
GemvShape gemv_pick(GemmEpi, int, int) { return GemvShape{8, 1, 2, 1}; }
hipError_t launch_gemv(GemmEpi, const GemvArgs&, GemvShape, const Exec&) { return hipSuccess; }
hipError_t launch_pack(const bf16_t*, const bf16_t*, bf16_t*, int64_t, int, int, hipStream_t) { return hipSuccess; }
hipError_t launch_embed(const EmbedArgs&, const Exec&) { return hipSuccess; }
hipError_t launch_rope_stage(const RopeStageArgs&, const Exec&) { return hipSuccess; }
hipError_t launch_rope_table(float*, int64_t, int, double, hipStream_t) { return hipSuccess; }
hipError_t launch_kv_import(const KvCopyArgs&, hipStream_t) { return hipSuccess; }
hipError_t launch_kv_export(const KvCopyArgs&, hipStream_t) { return hipSuccess; }
hipError_t launch_attention_split(const AttnArgs&, const Exec&) { return hipSuccess; }
hipError_t launch_attention_merge(const AttnArgs&, const Exec&) { return hipSuccess; }
bool fused_plan(FwdArgs&, int, int64_t) { return false; }
hipError_t launch_fused_forward(const FwdArgs&, int, const Exec&) { return hipSuccess; }
bool layer_xcd_fits(const sbd_model_config&, int, int, int) { return false; }
hipError_t launch_layer_attn(const LayerXArgs&, bool, const Exec&) { return hipSuccess; }
hipError_t launch_layer_mlp(const LayerXArgs&, bool, const Exec&) { return hipSuccess; }
hipError_t launch_layer_finalize(const FinalizeArgs&, const Exec&) { return hipSuccess; }
hipError_t launch_eb_partial(const EbArgs&, const Exec&) { return hipSuccess; }
hipError_t launch_eb_select(const EbArgs&, bool, const Exec&) { return hipSuccess; }
hipError_t launch_eb_merge(const EbArgs&, const Exec&) { return hipSuccess; }
hipError_t launch_pack_fp8(const fp8_t*, const fp8_t*, fp8_t*, int64_t, int, int, hipStream_t) { return hipSuccess; }
hipError_t launch_pack_fp8_widen(const fp8_t*, const fp8_t*, int, int, bf16_t*, int64_t, int, int, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_xcd_probe(int*, int, hipStream_t) { return hipSuccess; }
hipError_t launch_stream_probe(const void*, int64_t, uint32_t*, int, hipStream_t) { return hipSuccess; }

static double g_scratch[(int64_t)kNoAllocRows * kNoAllocChunks * 3 + (int64_t)kNoAllocRows * kNoAllocChunks / 2];
hipError_t eb_noalloc_scratch(double** part, int32_t** part_arg) {
  *part = g_scratch;
  *part_arg = reinterpret_cast<int32_t*>(g_scratch + (int64_t)kNoAllocRows * kNoAllocChunks * 3);
  return hipSuccess;
}

}  // namespace sbd
