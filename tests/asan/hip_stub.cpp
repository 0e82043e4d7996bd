// A stand-in for the HIP runtime, for a CPU-only build of libsagips's host code
// under AddressSanitizer and UndefinedBehaviorSanitizer: one device that reports
// itself as gfx950 with 256 compute units, hipMalloc backed by host malloc (so
// the sanitizer tracks every workspace the library allocates), and kernel
// launches that run nothing but check the launch shape the library asks for.
// Device pointers handed to the library are never dereferenced by its host code;
// the stub keeps it that way by not running any kernel.
#include <hip/hip_runtime_api.h>

#include <atomic>
#include <cstdio>
#include <cstdlib>
#include <cstring>

namespace {
const char* g_arch = "gfx950";
std::atomic<long> g_launches{0}, g_bad_launches{0}, g_live_events{0}, g_live_allocs{0};
size_t g_malloc_limit = (size_t)1 << 31;   // larger requests fail, as a full device would
unsigned char* g_symbol_block = nullptr;   // backs hipGetSymbolAddress
thread_local dim3 g_grid, g_block;
thread_local size_t g_shmem = 0;
}  // namespace

extern "C" {
void stub_set_arch(const char* arch) { g_arch = arch; }
long stub_launches() { return g_launches.load(); }
long stub_bad_launches() { return g_bad_launches.load(); }
long stub_live_events() { return g_live_events.load(); }
long stub_live_allocs() { return g_live_allocs.load(); }

void** __hipRegisterFatBinary(const void*) {
  static void* handle = nullptr;
  return &handle;
}
void __hipUnregisterFatBinary(void**) {}
void __hipRegisterFunction(void**, const void*, char*, const char*, unsigned int, void*, void*, dim3*, dim3*, int*) {}
void __hipRegisterVar(void**, void*, char*, char*, int, size_t, int, int) {}
}

hipError_t __hipPushCallConfiguration(dim3 grid, dim3 block, size_t shmem, hipStream_t) {
  g_grid = grid;
  g_block = block;
  g_shmem = shmem;
  return hipSuccess;
}
hipError_t __hipPopCallConfiguration(dim3* grid, dim3* block, size_t* shmem, hipStream_t* stream) {
  *grid = g_grid;
  *block = g_block;
  *shmem = g_shmem;
  *stream = nullptr;
  return hipSuccess;
}

hipError_t hipLaunchKernel(const void* fn, dim3 grid, dim3 block, void**, size_t shmem, hipStream_t) {
  g_launches++;
  const unsigned long long threads = (unsigned long long)block.x * block.y * block.z;
  const bool ok = fn && grid.x >= 1 && grid.y >= 1 && grid.z >= 1 && grid.x <= 0x7fffffffu && grid.y <= 65535 &&
                  grid.z <= 65535 && threads >= 1 && threads <= 1024 && shmem <= 160 * 1024 &&
                  (unsigned long long)grid.x * block.x < (1ull << 32);
  if (!ok) {
    g_bad_launches++;
    fprintf(stderr, "stub: bad launch grid (%u,%u,%u) block (%u,%u,%u) shmem %zu\n", grid.x, grid.y, grid.z,
            block.x, block.y, block.z, shmem);
  }
  return hipSuccess;
}

hipError_t hipGetDeviceCount(int* n) {
  *n = 1;
  return hipSuccess;
}
hipError_t hipGetDevice(int* d) {
  *d = 0;
  return hipSuccess;
}
hipError_t hipSetDevice(int d) { return d == 0 ? hipSuccess : hipErrorInvalidDevice; }
hipError_t hipGetDevicePropertiesR0600(hipDeviceProp_tR0600* p, int d) {
  if (d != 0) return hipErrorInvalidDevice;
  memset(p, 0, sizeof(*p));
  strncpy(p->gcnArchName, g_arch, sizeof(p->gcnArchName) - 1);
  p->multiProcessorCount = 256;
  return hipSuccess;
}
hipError_t hipMalloc(void** p, size_t n) {
  if (n > g_malloc_limit) {
    *p = nullptr;
    return hipErrorOutOfMemory;
  }
  *p = malloc(n ? n : 1);
  if (!*p) return hipErrorOutOfMemory;
  g_live_allocs++;
  return hipSuccess;
}
hipError_t hipFree(void* p) {
  if (p) {
    g_live_allocs--;
    free(p);
  }
  return hipSuccess;
}
hipError_t hipGetLastError() { return hipSuccess; }
const char* hipGetErrorString(hipError_t) { return "stub error"; }
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
hipError_t hipStreamWaitEvent(hipStream_t, hipEvent_t e, unsigned int) { return e ? hipSuccess : hipErrorInvalidValue; }
hipError_t hipEventCreate(hipEvent_t* e) {
  *e = reinterpret_cast<hipEvent_t>(new int(0));
  g_live_events++;
  return hipSuccess;
}
hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned) { return hipEventCreate(e); }
hipError_t hipEventDestroy(hipEvent_t e) {
  if (!e) return hipErrorInvalidValue;
  delete reinterpret_cast<int*>(e);
  g_live_events--;
  return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t e, hipStream_t) { return e ? hipSuccess : hipErrorInvalidValue; }
hipError_t hipEventElapsedTime(float* ms, hipEvent_t a, hipEvent_t b) {
  *ms = 0.0f;
  return (a && b) ? hipSuccess : hipErrorInvalidValue;
}
hipError_t hipGetSymbolAddress(void** p, const void* sym) {
  if (!sym) return hipErrorInvalidSymbol;
  if (!g_symbol_block) g_symbol_block = static_cast<unsigned char*>(aligned_alloc(256, (size_t)64 << 20));
  *p = g_symbol_block;
  return hipSuccess;
}
