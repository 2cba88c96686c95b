// A host-memory stand-in for the HIP runtime and for the kernel launchers, so
// that the library's host API sources (api.cpp, fusion_api.cpp,
// kvproj_api.cpp) can be built with AddressSanitizer and UBSan and driven on a
// machine without a GPU.  "Device" memory is host memory, copies are memcpy,
// events and streams are no-ops, and a launcher only checks the parameters the
// host side hands it (the checks a kernel relies on) and counts the launch.
// The validate launchers report "no violation".
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "fusion_common.h"
#include "kvproj_common.h"
#include "kvshot_common.h"

int g_launches = 0;
int g_bad_params = 0;

namespace {
void need(bool ok, const char* what) {
  if (!ok) {
    std::fprintf(stderr, "stub: bad launch parameter: %s\n", what);
    ++g_bad_params;
  }
}
}  // namespace

extern "C" {
hipError_t hipMalloc(void** p, size_t bytes) {
  if (!p) return hipErrorInvalidValue;
  *p = nullptr;
  if (posix_memalign(p, 256, bytes ? bytes : 1) != 0) return hipErrorOutOfMemory;
  return hipSuccess;
}
hipError_t hipFree(void* p) {
  std::free(p);
  return hipSuccess;
}
hipError_t hipMemcpy(void* dst, const void* src, size_t n, hipMemcpyKind) {
  std::memcpy(dst, src, n);
  return hipSuccess;
}
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t n, hipMemcpyKind, hipStream_t) {
  std::memcpy(dst, src, n);
  return hipSuccess;
}
hipError_t hipGetDevice(int* d) {
  *d = 0;
  return hipSuccess;
}
hipError_t hipSetDevice(int d) { return d == 0 ? hipSuccess : hipErrorInvalidDevice; }
hipError_t hipGetDevicePropertiesR0600(hipDeviceProp_tR0600* prop, int) {
  std::memset((void*)prop, 0, sizeof(*prop));
  prop->multiProcessorCount = 256;
  return hipSuccess;
}
hipError_t hipDeviceSynchronize() { return hipSuccess; }
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
hipError_t hipGetLastError() { return hipSuccess; }
hipError_t hipEventCreate(hipEvent_t* e) {
  *e = (hipEvent_t) new int(0);
  return hipSuccess;
}
hipError_t hipEventDestroy(hipEvent_t e) {
  delete (int*)e;
  return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t e, hipStream_t) { return e ? hipSuccess : hipErrorInvalidValue; }
hipError_t hipEventSynchronize(hipEvent_t e) { return e ? hipSuccess : hipErrorInvalidValue; }
hipError_t hipEventQuery(hipEvent_t e) { return e ? hipSuccess : hipErrorInvalidValue; }
hipError_t hipEventElapsedTime(float* ms, hipEvent_t a, hipEvent_t b) {
  if (!a || !b) return hipErrorInvalidValue;
  *ms = 0.01f;
  return hipSuccess;
}
// a __device__ array's host shadow stands for its device copy
hipError_t hipGetSymbolAddress(void** p, const void* symbol) {
  *p = const_cast<void*>(symbol);
  return hipSuccess;
}
void** __hipRegisterFatBinary(const void*) {
  static void* handle = nullptr;
  return &handle;
}
void __hipUnregisterFatBinary(void**) {}
void __hipRegisterVar(void**, void*, char*, char*, int, size_t, int, int) {}
}  // extern "C"

namespace kvshot {
int tall_waves_per_wg() { return 8; }
int tall_max_blocks() { return 512; }
int mfma_waves_per_wg(int kernel_row_tiles) { return kernel_row_tiles >= 8 ? 8 : 4; }
int mfma_key_streams(int kernel_row_tiles) { return mfma_waves_per_wg(kernel_row_tiles) / kernel_row_tiles; }
int mfma_wgs_per_cu(int) { return 1; }
int mfma_kernel_row_tiles(int row_tiles) { return row_tiles > 8 ? 8 : row_tiles; }

// `kernel`: an attention kernel launch, which reads the split plan (the gather and validate
// kernels only address pages)
static void check_attn(const AttnParams& p, bool kernel = true) {
  need(p.batch >= 1 && p.hkv >= 1 && p.hq >= p.hkv, "batch / heads");
  need(p.splits >= 1, "splits");
  need(p.splits == 1 || (p.part_o && p.part_ml), "split partials");
  need(!kernel || !p.balanced || (p.items > p.batch && p.seq_splits && p.min_chunk >= 1), "balanced schedule");
  need(p.page_table && p.ctx_lens, "tables");
  ++g_launches;
}
hipError_t launch_attn_mfma(const AttnParams& p, int kernel_row_tiles, hipStream_t) {
  need(kernel_row_tiles == 1 || kernel_row_tiles == 2 || kernel_row_tiles == 4 || kernel_row_tiles == 8, "row tiles");
  check_attn(p);
  return hipSuccess;
}
hipError_t launch_attn_tall(const AttnParams& p, hipStream_t) {
  check_attn(p);
  return hipSuccess;
}
hipError_t launch_attn_generic(const AttnParams& p, int, hipStream_t) {
  check_attn(p);
  return hipSuccess;
}
hipError_t launch_combine(const CombineParams& p, hipStream_t) {
  need(p.splits >= 2, "combine splits");
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_gather_kv(const AttnParams& p, int, void* k, void* v, int, hipStream_t) {
  need(k && v, "gather outputs");
  check_attn(p, false);
  return hipSuccess;
}
hipError_t launch_tree_mask(const int32_t* parents, int batch, int n, uint64_t* anc, int32_t* depth, hipStream_t) {
  need(parents && anc && depth && batch >= 1 && n >= 1 && n <= 64, "tree mask");
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_validate(const AttnParams&, int, int32_t* flag, hipStream_t) {
  *flag = 0x7fffffff;
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_stream_read(const void* src, int64_t bytes, void* sink, int blocks, hipStream_t) {
  need(src && sink && bytes > 0 && blocks > 0, "stream read");
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_mfma_rate(int blocks, int iters, void* sink, hipStream_t) {
  need(sink && blocks > 0 && iters > 0, "mfma rate");
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_fusion(const FusionParams& p, hipStream_t) {
  need(p.tile_tokens == 64 || p.tile_tokens == 128, "fusion tile");
  need(p.m_tiles * p.tile_tokens >= p.tokens && (p.m_tiles - 1) * p.tile_tokens < p.tokens, "fusion token tiles");
  need(p.splits >= 1 && p.kparts >= 1 && p.splits % p.kparts == 0 && (4 * p.kparts) % p.splits == 0, "fusion splits");
  need((p.d / p.kparts) % 64 == 0, "fusion reduction parts");
  need(p.tile_tokens == 64 || p.kparts == p.splits, "128-token tiles split the index range");
  need(p.splits == 1 || p.part, "fusion partials");
  need(p.w_packed || (p.w_g && p.w_delta), "fusion weights");
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_fusion_combine(const FusionParams&, hipStream_t) {
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_fusion_pack(const uint16_t* w_g, const uint16_t* w_delta, uint16_t* packed, int d, hipStream_t) {
  need(w_g && w_delta && packed && d > 0, "fusion pack");
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_kvproj(const KvProjParams& p, hipStream_t) {
  need(p.splits >= 1 && (p.splits == 1 || p.part), "kvproj splits");
  need(p.work_items >= 1, "kvproj grid");
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_kvproj_combine(const KvProjParams& p, hipStream_t) {
  need(p.splits >= 2, "kvproj combine");
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_kvproj_direct(const KvProjParams& p, hipStream_t) {
  need(p.tile16 >= 1 && p.tile16 <= kProjDirectMaxTile16, "direct tile");
  need(p.work_items == 4 * p.hkv * p.n_tiles, "direct grid");
  need(p.n_tiles * 16 * p.tile16 >= p.n_tokens, "direct token tiles");
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_kvproj_validate(const KvProjParams&, int32_t* flag, hipStream_t) {
  *flag = 0x7fffffff;
  ++g_launches;
  return hipSuccess;
}
}  // namespace kvshot
