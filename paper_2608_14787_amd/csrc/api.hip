// Status strings, error reporting and device checks of the C ABI.
#include "sdd_internal.h"

#include <algorithm>

namespace sdd {

static thread_local std::string g_last_error;

void set_error(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
}

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(SDD_EHIP, "%s launch failed: %s", what, hipGetErrorString(e));
  return SDD_OK;
}

}  // namespace sdd

extern "C" const char* sdd_status_string(int status) {
  switch (status) {
    case SDD_OK: return "ok";
    case SDD_EINVAL: return "invalid argument";
    case SDD_ENOMEM: return "buffer too small or host allocation failed";
    case SDD_EHIP: return "HIP error";
    case SDD_ECAPACITY: return "capacity exceeded";
    case SDD_EUNSUPPORTED: return "unsupported configuration";
  }
  return "unknown status";
}

extern "C" const char* sdd_last_error(void) { return sdd::g_last_error.c_str(); }

extern "C" int sdd_device_ok(void) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return 0;
  return std::string(prop.gcnArchName).rfind("gfx950", 0) == 0 ? 1 : 0;
}

namespace {
__global__ void zero_words_kernel(uint32_t* p, size_t n) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = 0u;
}
}  // namespace

extern "C" int sdd_workspace_init(void* ws, size_t bytes, sdd_stream_t stream) {
  SDD_REQUIRE(ws != nullptr && bytes > 0, "NULL or empty workspace");
  SDD_REQUIRE((uintptr_t)ws % 16 == 0, "workspace must be 16-byte aligned");
  // a kernel, not hipMemsetAsync, so that the call may sit inside captured graphs
  const size_t words = bytes / 4;
  const int blocks = (int)std::min<size_t>(1024, (words + 255) / 256);
  hipLaunchKernelGGL(zero_words_kernel, dim3(blocks > 0 ? blocks : 1), dim3(256), 0,
                     reinterpret_cast<hipStream_t>(stream), reinterpret_cast<uint32_t*>(ws), words);
  return sdd::check_launch("zero_words_kernel");
}
