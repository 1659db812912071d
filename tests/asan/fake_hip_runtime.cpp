// A host-only stand-in for the HIP runtime, for the AddressSanitizer build of
// the library's host code on a machine without a GPU.  "Device" memory is
// host memory: copies are memcpy (so ASan checks every byte a table upload
// writes into a caller's workspace), events and graphs are tokens, and a
// kernel launch runs nothing but has its launch shape checked against the
// hardware limits (grid y/z <= 65535, x < 2^31, 1..1024 threads per block,
// <= 160 KiB of LDS).  Test infrastructure only.
#include <hip/hip_runtime_api.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>

extern "C" {

long long jn_fake_launches = 0;
long long jn_fake_graph_launches = 0;

static dim3 g_grid, g_block;
static size_t g_shm = 0;
static hipStream_t g_stream = nullptr;
static int g_capturing = 0;

struct FakeToken {
  int kind;
};

static void check_launch(dim3 grid, dim3 block, size_t shm) {
  const unsigned long long threads = (unsigned long long)block.x * block.y * block.z;
  if (grid.x < 1 || grid.x > 0x7fffffffu || grid.y < 1 || grid.y > 65535 || grid.z < 1 || grid.z > 65535 ||
      threads < 1 || threads > 1024 || shm > 160 * 1024) {
    std::fprintf(stderr, "bad launch shape: grid %u %u %u block %u %u %u lds %zu\n", grid.x, grid.y, grid.z,
                 block.x, block.y, block.z, shm);
    std::abort();
  }
}

void** __hipRegisterFatBinary(const void*) {
  static void* handle = nullptr;
  return &handle;
}
void __hipUnregisterFatBinary(void**) {}
void __hipRegisterFunction(void**, const void*, char*, const char*, unsigned int, void*, void*, void*, void*,
                           int*) {}
void __hipRegisterVar(void**, void*, char*, char*, int, size_t, int, int) {}

hipError_t __hipPushCallConfiguration(dim3 grid, dim3 block, size_t shm, hipStream_t stream) {
  g_grid = grid;
  g_block = block;
  g_shm = shm;
  g_stream = stream;
  return hipSuccess;
}
hipError_t __hipPopCallConfiguration(dim3* grid, dim3* block, size_t* shm, hipStream_t* stream) {
  *grid = g_grid;
  *block = g_block;
  *shm = g_shm;
  *stream = g_stream;
  return hipSuccess;
}
hipError_t hipLaunchKernel(const void* fn, dim3 grid, dim3 block, void** args, size_t shm, hipStream_t) {
  if (!fn || !args) std::abort();
  check_launch(grid, block, shm);
  ++jn_fake_launches;
  return hipSuccess;
}

hipError_t hipGetDevice(int* dev) {
  *dev = 0;
  return hipSuccess;
}
hipError_t hipDeviceGetAttribute(int* value, hipDeviceAttribute_t attr, int) {
  *value = attr == hipDeviceAttributeMultiprocessorCount ? 256 : 0;  // MI355X
  return hipSuccess;
}
hipError_t hipGetLastError(void) { return hipSuccess; }
const char* hipGetErrorString(hipError_t) { return "fake runtime error"; }

hipError_t hipEventCreate(hipEvent_t* e) {
  *e = reinterpret_cast<hipEvent_t>(new FakeToken{1});
  return hipSuccess;
}
hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned) { return hipEventCreate(e); }
hipError_t hipEventDestroy(hipEvent_t e) {
  delete reinterpret_cast<FakeToken*>(e);
  return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t e, hipStream_t) { return e ? hipSuccess : hipErrorInvalidValue; }
hipError_t hipEventSynchronize(hipEvent_t e) { return e ? hipSuccess : hipErrorInvalidValue; }
// every other query reports the work as still in flight, so callers' "not
// ready" paths (the staging ring growing) run under the sanitizer too
hipError_t hipEventQuery(hipEvent_t e) {
  static unsigned calls = 0;
  if (!e) return hipErrorInvalidValue;
  return (++calls & 1) ? hipErrorNotReady : hipSuccess;
}
hipError_t hipEventElapsedTime(float* ms, hipEvent_t a, hipEvent_t b) {
  if (!a || !b) return hipErrorInvalidValue;
  *ms = 0.f;
  return hipSuccess;
}

hipError_t hipHostMalloc(void** p, size_t n, unsigned int) {
  *p = std::malloc(n ? n : 1);
  return *p ? hipSuccess : hipErrorOutOfMemory;
}
hipError_t hipHostFree(void* p) {
  std::free(p);
  return hipSuccess;
}
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t n, hipMemcpyKind, hipStream_t) {
  if (n) std::memcpy(dst, src, n);
  return hipSuccess;
}
hipError_t hipGetSymbolAddress(void** p, const void* symbol) {
  *p = const_cast<void*>(symbol);
  return hipSuccess;
}

hipError_t hipStreamBeginCapture(hipStream_t s, hipStreamCaptureMode) {
  if (!s || g_capturing) return hipErrorInvalidValue;
  g_capturing = 1;
  return hipSuccess;
}
hipError_t hipStreamEndCapture(hipStream_t, hipGraph_t* g) {
  if (!g_capturing) return hipErrorInvalidValue;
  g_capturing = 0;
  *g = reinterpret_cast<hipGraph_t>(new FakeToken{2});
  return hipSuccess;
}
hipError_t hipGraphInstantiate(hipGraphExec_t* x, hipGraph_t g, hipGraphNode_t*, char*, size_t) {
  if (!g) return hipErrorInvalidValue;
  *x = reinterpret_cast<hipGraphExec_t>(new FakeToken{3});
  return hipSuccess;
}
hipError_t hipGraphLaunch(hipGraphExec_t x, hipStream_t) {
  if (!x) return hipErrorInvalidValue;
  ++jn_fake_graph_launches;
  return hipSuccess;
}
hipError_t hipGraphDestroy(hipGraph_t g) {
  delete reinterpret_cast<FakeToken*>(g);
  return hipSuccess;
}
hipError_t hipGraphExecDestroy(hipGraphExec_t x) {
  delete reinterpret_cast<FakeToken*>(x);
  return hipSuccess;
}

}  // extern "C"
