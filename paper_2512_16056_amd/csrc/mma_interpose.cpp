// Transparent interposition (Section 3.2, Transfer Task Interceptor): loaded
// with LD_PRELOAD, this library exports hipMemcpyAsync, hipMemcpy and
// hipMemcpyWithStream. A host<->device copy of at least MMA_INTERPOSE_MIN_BYTES
// (default 32 KiB) goes through libmma.so; everything else, and every copy that
// libmma refuses before any of it is enqueued (pageable host memory, another
// device), goes to the runtime's own function. The application is not changed
// and not relinked.
//
// Blocking copies (hipMemcpy, hipMemcpyWithStream) stay with the runtime unless
// MMA_INTERPOSE_SYNC=1. A blocking caller waits from the call to the copy's
// completion, and on one GPU that wait is not shorter through libmma at any
// size: its dummy-task kernel adds a kernel dispatch and completion round trip
// and a CU ramp-up that the copy engines' direct path does not have (call to
// return of hipStreamSynchronize on an idle stream, 32 KiB to 8 GiB: 0.41 to
// 0.999 of the runtime's speed). An asynchronous copy is judged on the stream,
// where the library is at or ahead of the runtime from 32 KiB up -- when the
// stream has work pending. On a stream with nothing pending the runtime's copy
// engine starts sooner than a kernel and one engine fills the link, so the
// runtime copy is the faster at every size measured (0.46 to 0.993 of its speed
// through libmma, 32 KiB to 8 GiB): such a copy stays with the runtime unless
// MMA_INTERPOSE_IDLE=1 (the fallback to the native copy of Section 3.2, decided
// by the stream's state as well as the size).
//
// Failures are never silent, and a copy is never issued twice over the same
// bytes while part of it may still be moving:
//   - a synchronous copy (hipMemcpy, hipMemcpyWithStream) that libmma reports
//     failed and retired -- no path writes its destination any more -- is
//     re-issued with the runtime's copy, and the failure is written to stderr;
//     one that is not retired within libmma's limit returns hipErrorUnknown;
//   - an asynchronous copy fails after its call has returned, so libmma keeps
//     the failure (sticky) and the next interposed call reports it: that call
//     returns hipErrorUnknown and writes the failure to stderr, and libmma's
//     sticky state is cleared so that later copies go through it again.
//
// The library links neither the HIP runtime nor libmma.so: both are resolved
// at the first intercepted call, so the process keeps using the HIP runtime it
// loads itself. libmma.so is taken from MMA_LIB, else from this library's
// directory; it is initialised on the device current at the first call (the
// usual MMA_* environment applies) and finalised at exit.
#include <dlfcn.h>
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <mutex>
#include <string>

#include "../../include/mma.h"

namespace {

typedef hipError_t (*async_fn)(void*, const void*, size_t, hipMemcpyKind, hipStream_t);
typedef hipError_t (*sync_fn)(void*, const void*, size_t, hipMemcpyKind);
typedef hipError_t (*get_device_fn)(int*);
typedef hipError_t (*attrs_fn)(hipPointerAttribute_t*, const void*);
typedef hipError_t (*query_fn)(hipStream_t);

struct Real {
  async_fn memcpy_async = nullptr;
  sync_fn memcpy = nullptr;
  async_fn memcpy_with_stream = nullptr;
  get_device_fn get_device = nullptr;
  attrs_fn pointer_attributes = nullptr;
  query_fn stream_query = nullptr;
};

struct Lib {
  mma_status_t (*init)(int, const mma_config_t*) = nullptr;
  mma_status_t (*finalize)(void) = nullptr;
  mma_status_t (*memcpy_async)(void*, const void*, uint64_t, int32_t, void*) = nullptr;
  mma_status_t (*memcpy_stream)(void*, const void*, uint64_t, int32_t, void*, int32_t*) = nullptr;
  mma_status_t (*clear_error)(void) = nullptr;
  const char* (*last_error)(void) = nullptr;
};

std::once_flag g_real_once, g_lib_once;
Real g_real;
Lib g_lib;
bool g_on = false;  // libmma is loaded and initialised
int g_dev = -1;
uint64_t g_min_bytes = 32 * 1024;
bool g_sync = false;  // blocking copies through libmma too (MMA_INTERPOSE_SYNC=1)
bool g_idle = false;  // asynchronous copies on a stream with nothing pending too (MMA_INTERPOSE_IDLE=1)

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
  g_real.stream_query = reinterpret_cast<query_fn>(runtime_symbol(rt, "hipStreamQuery"));
}

void finalize_at_exit() {
  if (g_on && g_lib.finalize) g_lib.finalize();
}

void load_lib() {
  if (!g_real.get_device || g_real.get_device(&g_dev) != hipSuccess) return;
  const char* env_min = getenv("MMA_INTERPOSE_MIN_BYTES");
  if (env_min && *env_min) g_min_bytes = strtoull(env_min, nullptr, 0);
  const char* env_sync = getenv("MMA_INTERPOSE_SYNC");
  g_sync = env_sync && strtoull(env_sync, nullptr, 0) != 0;
  const char* env_idle = getenv("MMA_INTERPOSE_IDLE");
  g_idle = env_idle && strtoull(env_idle, nullptr, 0) != 0;
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
  g_lib.memcpy_stream = reinterpret_cast<decltype(g_lib.memcpy_stream)>(dlsym(h, "mma_memcpy_stream"));
  g_lib.clear_error = reinterpret_cast<decltype(g_lib.clear_error)>(dlsym(h, "mma_clear_error"));
  g_lib.last_error = reinterpret_cast<decltype(g_lib.last_error)>(dlsym(h, "mma_last_error"));
  if (!g_lib.init || !g_lib.finalize || !g_lib.memcpy_async || !g_lib.memcpy_stream || !g_lib.clear_error ||
      !g_lib.last_error)
    return;
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

// An earlier asynchronous copy failed (libmma's sticky state): report it as
// this call's error and clear it, so that later copies go through libmma again.
hipError_t report_earlier_failure(const char* api) {
  fprintf(stderr, "[mma_interpose] %s: an earlier copy through libmma failed, its destination may be incomplete: "
                  "%s\n", api, g_lib.last_error());
  g_lib.clear_error();
  return hipErrorUnknown;
}

// A blocking copy through libmma on `stream`; falls back to the runtime copy
// only when nothing of the libmma copy is in flight.
hipError_t sync_copy(const char* api, void* dst, const void* src, size_t bytes, hipMemcpyKind kind, int dir,
                     hipStream_t stream, bool* use_runtime) {
  int32_t outcome = MMA_COPY_NOT_ENQUEUED;
  const mma_status_t s = g_lib.memcpy_stream(dst, src, bytes, dir, stream, &outcome);
  *use_runtime = false;
  if (s == MMA_OK) return hipSuccess;
  if (outcome == MMA_COPY_NOT_ENQUEUED) {
    if (s == MMA_ERR_TRANSFER_FAILED) return report_earlier_failure(api);
    *use_runtime = true;  // refused: the runtime copies it
    return hipSuccess;
  }
  if (outcome == MMA_COPY_RETIRED) {  // this copy failed, and nothing writes its destination any more
    fprintf(stderr, "[mma_interpose] %s: copy of %zu bytes failed in libmma (%s); copied again by the runtime\n",
            api, bytes, g_lib.last_error());
    g_lib.clear_error();
    *use_runtime = true;
    return hipSuccess;
  }
  fprintf(stderr, "[mma_interpose] %s: copy of %zu bytes (kind %d) did not finish in libmma (%s)\n", api, bytes,
          static_cast<int>(kind), g_lib.last_error());
  return hipErrorUnknown;  // parts may still be moving: a second copy could interleave with them
}

}  // namespace

extern "C" {

hipError_t hipMemcpyAsync(void* dst, const void* src, size_t bytes, hipMemcpyKind kind, hipStream_t stream) {
  int dir = route(dst, src, bytes, kind);
  // Nothing pending on the stream: the runtime's copy is the faster one. An
  // earlier asynchronous failure is still reported here (a zero-byte call
  // returns libmma's sticky state and enqueues nothing).
  if (dir >= 0 && !g_idle && g_real.stream_query && g_real.stream_query(stream) == hipSuccess) {
    if (g_lib.memcpy_async(nullptr, nullptr, 0, dir, stream) == MMA_ERR_TRANSFER_FAILED)
      return report_earlier_failure("hipMemcpyAsync");
    dir = -1;
  }
  if (dir >= 0) {
    const mma_status_t s = g_lib.memcpy_async(dst, src, bytes, dir, stream);
    if (s == MMA_OK) return hipSuccess;
    if (s == MMA_ERR_TRANSFER_FAILED) return report_earlier_failure("hipMemcpyAsync");
    // refused, or its launch failed: nothing of it is in flight
  }
  if (!g_real.memcpy_async) return hipErrorNotSupported;
  return g_real.memcpy_async(dst, src, bytes, kind, stream);
}

hipError_t hipMemcpy(void* dst, const void* src, size_t bytes, hipMemcpyKind kind) {
  const int dir = route(dst, src, bytes, kind);
  if (dir >= 0 && g_sync) {
    bool use_runtime = false;
    const hipError_t e = sync_copy("hipMemcpy", dst, src, bytes, kind, dir, nullptr, &use_runtime);
    if (!use_runtime) return e;
  }
  if (!g_real.memcpy) return hipErrorNotSupported;
  return g_real.memcpy(dst, src, bytes, kind);
}

// Synchronous with respect to the host, ordered on `stream`.
hipError_t hipMemcpyWithStream(void* dst, const void* src, size_t bytes, hipMemcpyKind kind, hipStream_t stream) {
  const int dir = route(dst, src, bytes, kind);
  if (dir >= 0 && g_sync) {
    bool use_runtime = false;
    const hipError_t e = sync_copy("hipMemcpyWithStream", dst, src, bytes, kind, dir, stream, &use_runtime);
    if (!use_runtime) return e;
  }
  if (!g_real.memcpy_with_stream) return hipErrorNotSupported;
  return g_real.memcpy_with_stream(dst, src, bytes, kind, stream);
}

}  // extern "C"
