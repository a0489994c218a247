// Shared tensor store: device allocations that one process owns and other
// processes on the same GPU map zero-copy through IPC handles, so that an
// engine can build a stage over weights and KV space it did not load
// (Sec. 5.2, "Shared Tensor Store"). The store side allocates and exports;
// the engine side attaches and detaches. Every allocation is one hipMalloc
// of less than 2 GiB and is exported as a whole, so a handle always maps
// exactly one allocation, from its base.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>

#include "../../include/stage.h"
#include "kernels.hpp"

namespace {

// Store errors share the thread-local message of the stage entry points.
stage_status store_fail(stage_status code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  stage_k::set_error(buf);
  return code;
}

static_assert(sizeof(hipIpcMemHandle_t) == sizeof(stage_ipc_handle),
              "stage_ipc_handle must hold a hipIpcMemHandle_t");

}  // namespace

extern "C" {

stage_status stage_store_alloc(size_t bytes, void** dev, stage_ipc_handle* handle) {
  if (!dev || !handle) return store_fail(STAGE_ERR_INVALID_ARG, "dev/handle is NULL");
  *dev = nullptr;
  if (bytes == 0) return store_fail(STAGE_ERR_INVALID_ARG, "store allocation of 0 bytes");
  if (bytes >= STAGE_STORE_MAX_BYTES)
    return store_fail(STAGE_ERR_CAPACITY, "store allocation of %zu bytes: each must be below %zu",
                      bytes, (size_t)STAGE_STORE_MAX_BYTES);
  void* p = nullptr;
  hipError_t e = hipMalloc(&p, bytes);
  if (e != hipSuccess)
    return store_fail(STAGE_ERR_DEVICE, "hipMalloc(%zu): %s", bytes, hipGetErrorString(e));
  if ((e = hipMemset(p, 0, bytes)) != hipSuccess) {
    (void)hipFree(p);
    return store_fail(STAGE_ERR_DEVICE, "hipMemset: %s", hipGetErrorString(e));
  }
  hipIpcMemHandle_t h;
  if ((e = hipIpcGetMemHandle(&h, p)) != hipSuccess) {
    (void)hipFree(p);
    return store_fail(STAGE_ERR_DEVICE, "hipIpcGetMemHandle: %s", hipGetErrorString(e));
  }
  std::memcpy(handle->bytes, &h, sizeof h);
  *dev = p;
  return STAGE_OK;
}

stage_status stage_store_free(void* dev) {
  if (!dev) return STAGE_OK;
  hipError_t e = hipFree(dev);
  if (e != hipSuccess) return store_fail(STAGE_ERR_DEVICE, "hipFree: %s", hipGetErrorString(e));
  return STAGE_OK;
}

stage_status stage_store_write(void* dst, const void* src, size_t bytes, void* stream) {
  if (!dst || !src) return store_fail(STAGE_ERR_INVALID_ARG, "dst/src is NULL");
  hipError_t e = hipMemcpyAsync(dst, src, bytes, hipMemcpyDefault, (hipStream_t)stream);
  if (e != hipSuccess)
    return store_fail(STAGE_ERR_DEVICE, "hipMemcpyAsync: %s", hipGetErrorString(e));
  return STAGE_OK;
}

stage_status stage_store_attach(const stage_ipc_handle* handle, void** dev) {
  if (!handle || !dev) return store_fail(STAGE_ERR_INVALID_ARG, "handle/dev is NULL");
  *dev = nullptr;
  hipIpcMemHandle_t h;
  std::memcpy(&h, handle->bytes, sizeof h);
  void* p = nullptr;
  hipError_t e = hipIpcOpenMemHandle(&p, h, hipIpcMemLazyEnablePeerAccess);
  if (e != hipSuccess)
    return store_fail(STAGE_ERR_DEVICE, "hipIpcOpenMemHandle: %s", hipGetErrorString(e));
  *dev = p;
  return STAGE_OK;
}

stage_status stage_store_detach(void* dev) {
  if (!dev) return STAGE_OK;
  hipError_t e = hipIpcCloseMemHandle(dev);
  if (e != hipSuccess)
    return store_fail(STAGE_ERR_DEVICE, "hipIpcCloseMemHandle: %s", hipGetErrorString(e));
  return STAGE_OK;
}

}  // extern "C"
