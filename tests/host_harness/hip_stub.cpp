// hip_stub.cpp -- a stand-in for the HIP runtime, linked into host-only builds of libsparda's
// sources so that their host code (argument validation, workspace sizing, launch planning) runs
// under AddressSanitizer and UndefinedBehaviorSanitizer on a machine without a GPU.  Nothing runs
// on a device: every kernel launch is recorded and its configuration checked against the limits
// a real launch must respect (grid >= 1 per axis, grid.y and grid.z <= 65535, grid x block
// < 2^32 work items per axis, 1..1024 threads per workgroup, dynamic LDS <= 160 KiB).
// Pinned host pools are simulated by ranges the harness registers.
#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "sparda.h"

namespace {
struct Range {
  uintptr_t base;
  size_t size;
};
std::vector<Range> g_host;
long g_launches = 0, g_bad_launches = 0;
dim3 g_grid, g_block;
size_t g_shmem = 0;
hipStream_t g_stream = nullptr;

const Range* find_range(const void* p) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(p);
  for (const Range& r : g_host)
    if (a >= r.base && a < r.base + r.size) return &r;
  return nullptr;
}
}  // namespace

extern "C" {

// ---- harness controls ---------------------------------------------------------------------------
void stub_register_host(const void* p, size_t bytes) { g_host.push_back({reinterpret_cast<uintptr_t>(p), bytes}); }
void stub_clear_host(void) { g_host.clear(); }
long stub_launches(void) { return g_launches; }
long stub_bad_launches(void) { return g_bad_launches; }

// ---- the runtime calls the library makes ------------------------------------------------------
hipError_t hipGetLastError(void) { return hipSuccess; }
const char* hipGetErrorString(hipError_t) { return "stub HIP error"; }
hipError_t hipGetDevice(int* device) {
  *device = 0;
  return hipSuccess;
}
hipError_t hipGetSymbolAddress(void** dev_ptr, const void*) {
  static void* scratch = std::calloc(1, SPARDA_NOALLOC_SCRATCH_BYTES);
  *dev_ptr = scratch;
  return scratch ? hipSuccess : hipErrorOutOfMemory;
}
hipError_t hipPointerGetAttributes(hipPointerAttribute_t* attr, const void* p) {
  const Range* r = find_range(p);
  if (!r) return hipErrorInvalidValue;
  attr->type = hipMemoryTypeHost;
  attr->device = 0;
  attr->devicePointer = const_cast<void*>(p);
  attr->hostPointer = const_cast<void*>(p);
  attr->isManaged = 0;
  attr->allocationFlags = 0;
  return hipSuccess;
}
hipError_t hipMemGetAddressRange(hipDeviceptr_t* base, size_t* size, hipDeviceptr_t p) {
  const Range* r = find_range(p);
  if (!r) return hipErrorInvalidValue;
  *base = reinterpret_cast<hipDeviceptr_t>(r->base);
  *size = r->size;
  return hipSuccess;
}
hipError_t __hipPushCallConfiguration(dim3 grid, dim3 block, size_t shmem, hipStream_t stream) {
  g_grid = grid;
  g_block = block;
  g_shmem = shmem;
  g_stream = stream;
  return hipSuccess;
}
hipError_t __hipPopCallConfiguration(dim3* grid, dim3* block, size_t* shmem, hipStream_t* stream) {
  *grid = g_grid;
  *block = g_block;
  *shmem = g_shmem;
  *stream = g_stream;
  return hipSuccess;
}
hipError_t hipLaunchKernel(const void*, dim3 grid, dim3 block, void**, size_t shmem, hipStream_t) {
  ++g_launches;
  const uint64_t threads = (uint64_t)block.x * block.y * block.z;
  const bool ok = grid.x >= 1 && grid.y >= 1 && grid.z >= 1 && grid.y <= 65535 && grid.z <= 65535 &&
                  threads >= 1 && threads <= 1024 && (uint64_t)grid.x * block.x < (1ull << 32) &&
                  shmem <= 160 * 1024;
  if (!ok) {
    ++g_bad_launches;
    std::fprintf(stderr, "bad launch: grid (%u, %u, %u) block (%u, %u, %u) lds %zu\n", grid.x, grid.y, grid.z,
                 block.x, block.y, block.z, shmem);
  }
  return hipSuccess;
}
void** __hipRegisterFatBinary(const void*) {
  static void* handle = nullptr;
  return &handle;
}
void __hipRegisterFunction(void**, const void*, char*, const char*, unsigned int, void*, void*, void*, void*, int*) {}
void __hipRegisterVar(void**, void*, char*, char*, int, size_t, int, int) {}
void __hipUnregisterFatBinary(void**) {}

}  // extern "C"
