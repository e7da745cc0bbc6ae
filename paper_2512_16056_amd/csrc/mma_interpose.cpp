// Transparent interposition (Section 3.2, Transfer Task Interceptor): loaded
// with LD_PRELOAD, this library exports hipMemcpyAsync, hipMemcpy and
// hipMemcpyWithStream. A host<->device copy of at least MMA_INTERPOSE_MIN_BYTES
// (default 32 KiB, where the multipath copy starts to beat one runtime copy on
// MI355X) goes through libmma.so; everything else, and every copy that libmma
// refuses (pageable host memory, another device, a sticky earlier failure),
// goes to the runtime's own function. The application is not changed and not
// relinked.
//
// The library links neither the HIP runtime nor libmma.so: both are resolved
// at the first intercepted call, so the process keeps using the HIP runtime it
// loads itself. libmma.so is taken from MMA_LIB, else from this library's
// directory; it is initialised on the device current at the first call (the
// usual MMA_* environment applies) and finalised at exit.
#include <dlfcn.h>
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdlib.h>

#include <mutex>
#include <string>

#include "../../include/mma.h"

namespace {

typedef hipError_t (*async_fn)(void*, const void*, size_t, hipMemcpyKind, hipStream_t);
typedef hipError_t (*sync_fn)(void*, const void*, size_t, hipMemcpyKind);
typedef hipError_t (*get_device_fn)(int*);
typedef hipError_t (*attrs_fn)(hipPointerAttribute_t*, const void*);
typedef hipError_t (*stream_sync_fn)(hipStream_t);

struct Real {
  async_fn memcpy_async = nullptr;
  sync_fn memcpy = nullptr;
  async_fn memcpy_with_stream = nullptr;
  get_device_fn get_device = nullptr;
  attrs_fn pointer_attributes = nullptr;
  stream_sync_fn stream_synchronize = nullptr;
};

struct Lib {
  mma_status_t (*init)(int, const mma_config_t*) = nullptr;
  mma_status_t (*finalize)(void) = nullptr;
  mma_status_t (*memcpy_async)(void*, const void*, uint64_t, int32_t, void*) = nullptr;
  mma_status_t (*memcpy)(void*, const void*, uint64_t, int32_t) = nullptr;
};

std::once_flag g_real_once, g_lib_once;
Real g_real;
Lib g_lib;
bool g_on = false;  // libmma is loaded and initialised
int g_dev = -1;
uint64_t g_min_bytes = 32 * 1024;

// The runtime's own functions. A program that links the HIP runtime has it in
// the global scope (RTLD_NEXT finds it); Python extensions load it with
// RTLD_LOCAL, so it is then looked up by its soname among the loaded objects.
void* runtime_symbol(void* rt, const char* name) {
  if (rt) {
    if (void* f = dlvsym(rt, name, "hip_4.2")) return f;  // the version programs built for HIP 4.2+ bind
    if (void* f = dlsym(rt, name)) return f;
  }
  return dlsym(RTLD_NEXT, name);
}

void resolve_real() {
  void* rt = dlopen("libamdhip64.so.7", RTLD_NOW | RTLD_NOLOAD);
  if (!rt) rt = dlopen("libamdhip64.so", RTLD_NOW | RTLD_NOLOAD);
  g_real.memcpy_async = reinterpret_cast<async_fn>(runtime_symbol(rt, "hipMemcpyAsync"));
  g_real.memcpy = reinterpret_cast<sync_fn>(runtime_symbol(rt, "hipMemcpy"));
  g_real.memcpy_with_stream = reinterpret_cast<async_fn>(runtime_symbol(rt, "hipMemcpyWithStream"));
  g_real.get_device = reinterpret_cast<get_device_fn>(runtime_symbol(rt, "hipGetDevice"));
  g_real.pointer_attributes = reinterpret_cast<attrs_fn>(runtime_symbol(rt, "hipPointerGetAttributes"));
  g_real.stream_synchronize = reinterpret_cast<stream_sync_fn>(runtime_symbol(rt, "hipStreamSynchronize"));
}

void finalize_at_exit() {
  if (g_on && g_lib.finalize) g_lib.finalize();
}

void load_lib() {
  if (!g_real.get_device || g_real.get_device(&g_dev) != hipSuccess) return;
  const char* env_min = getenv("MMA_INTERPOSE_MIN_BYTES");
  if (env_min && *env_min) g_min_bytes = strtoull(env_min, nullptr, 0);
  std::string path;
  const char* env_lib = getenv("MMA_LIB");
  if (env_lib && *env_lib) {
    path = env_lib;
  } else {
    Dl_info info;
    if (!dladdr(reinterpret_cast<void*>(&load_lib), &info) || !info.dli_fname) return;
    path = info.dli_fname;
    const size_t slash = path.rfind('/');
    path = (slash == std::string::npos ? std::string(".") : path.substr(0, slash)) + "/libmma.so";
  }
  void* h = dlopen(path.c_str(), RTLD_NOW | RTLD_GLOBAL);
  if (!h) return;
  g_lib.init = reinterpret_cast<decltype(g_lib.init)>(dlsym(h, "mma_init"));
  g_lib.finalize = reinterpret_cast<decltype(g_lib.finalize)>(dlsym(h, "mma_finalize"));
  g_lib.memcpy_async = reinterpret_cast<decltype(g_lib.memcpy_async)>(dlsym(h, "mma_memcpy_async"));
  g_lib.memcpy = reinterpret_cast<decltype(g_lib.memcpy)>(dlsym(h, "mma_memcpy"));
  if (!g_lib.init || !g_lib.finalize || !g_lib.memcpy_async || !g_lib.memcpy) return;
  const mma_status_t s = g_lib.init(g_dev, nullptr);
  if (s != MMA_OK && s != MMA_ERR_ALREADY_INITIALIZED) return;
  g_on = true;
  atexit(finalize_at_exit);
}

// Direction for libmma, or -1 to leave the copy to the runtime.
int route(void* dst, const void* src, size_t bytes, hipMemcpyKind kind) {
  std::call_once(g_real_once, resolve_real);
  if (bytes < g_min_bytes) return -1;
  if (kind != hipMemcpyHostToDevice && kind != hipMemcpyDeviceToHost && kind != hipMemcpyDefault) return -1;
  std::call_once(g_lib_once, load_lib);
  if (!g_on) return -1;
  int dev = -1;
  if (g_real.get_device(&dev) != hipSuccess || dev != g_dev) return -1;
  if (kind == hipMemcpyHostToDevice) return MMA_H2D;
  if (kind == hipMemcpyDeviceToHost) return MMA_D2H;
  if (!g_real.pointer_attributes) return -1;
  hipPointerAttribute_t a{}, b{};
  if (g_real.pointer_attributes(&a, src) != hipSuccess || g_real.pointer_attributes(&b, dst) != hipSuccess)
    return -1;
  if (a.type == hipMemoryTypeHost && b.type == hipMemoryTypeDevice) return MMA_H2D;
  if (a.type == hipMemoryTypeDevice && b.type == hipMemoryTypeHost) return MMA_D2H;
  return -1;
}

}  // namespace

extern "C" {

hipError_t hipMemcpyAsync(void* dst, const void* src, size_t bytes, hipMemcpyKind kind, hipStream_t stream) {
  const int dir = route(dst, src, bytes, kind);
  if (dir >= 0 && g_lib.memcpy_async(dst, src, bytes, dir, stream) == MMA_OK) return hipSuccess;
  if (!g_real.memcpy_async) return hipErrorNotSupported;
  return g_real.memcpy_async(dst, src, bytes, kind, stream);
}

hipError_t hipMemcpy(void* dst, const void* src, size_t bytes, hipMemcpyKind kind) {
  const int dir = route(dst, src, bytes, kind);
  if (dir >= 0 && g_lib.memcpy(dst, src, bytes, dir) == MMA_OK) return hipSuccess;
  if (!g_real.memcpy) return hipErrorNotSupported;
  return g_real.memcpy(dst, src, bytes, kind);
}

// Synchronous with respect to the host, ordered on `stream`.
hipError_t hipMemcpyWithStream(void* dst, const void* src, size_t bytes, hipMemcpyKind kind, hipStream_t stream) {
  const int dir = route(dst, src, bytes, kind);
  if (dir >= 0 && g_real.stream_synchronize && g_lib.memcpy_async(dst, src, bytes, dir, stream) == MMA_OK)
    return g_real.stream_synchronize(stream);
  if (!g_real.memcpy_with_stream) return hipErrorNotSupported;
  return g_real.memcpy_with_stream(dst, src, bytes, kind, stream);
}

}  // extern "C"
