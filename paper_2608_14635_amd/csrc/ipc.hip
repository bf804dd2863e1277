// Cross-process retained state (kvr_ipc.h): HIP IPC memory handles of the
// owner's allocations, tagged with the owner's process id.  Host code only.
#include <hip/hip_runtime.h>
#include <signal.h>
#include <unistd.h>

#include <cerrno>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>

#include "kvr.h"
#include "kvr_ipc.h"

// the calling thread's error message, shared with the rest of the library
namespace kvr_err {
kv_status set(kv_status st, const char* fmt, ...);
kv_status clear();
}  // namespace kvr_err

namespace {

std::mutex g_mu;
std::map<void*, void*> g_opened;  // returned pointer -> mapped allocation base

static_assert(sizeof(hipIpcMemHandle_t) <= 64, "IPC handle size");

// Handles are limited to allocations below 2 GiB: opening a handle of a
// larger allocation has been seen not to return.
constexpr uint64_t IPC_MAX_ALLOCATION = 2ull << 30;

}  // namespace

extern "C" {

kv_status kv_ipc_export(const void* ptr, uint64_t bytes, kv_ipc_handle* out) {
  if (!ptr || !out || bytes == 0) return kvr_err::set(KV_EINVAL, "null pointer or zero size");
  std::memset(out, 0, sizeof *out);
  if (bytes >= IPC_MAX_ALLOCATION)
    return kvr_err::set(KV_EINVAL, "%llu bytes: handles are limited to allocations below 2 GiB",
                        (unsigned long long)bytes);
  hipPointerAttribute_t attr;
  hipError_t e = hipPointerGetAttributes(&attr, ptr);
  if (e != hipSuccess || attr.type != hipMemoryTypeDevice) {
    (void)hipGetLastError();
    return kvr_err::set(KV_EDEVICE, "pointer is not device memory known to HIP");
  }
  hipDeviceptr_t base = nullptr;
  size_t size = 0;
  e = hipMemGetAddressRange(&base, &size, const_cast<void*>(ptr));
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return kvr_err::set(KV_EDEVICE, "no allocation range for the pointer: %s", hipGetErrorString(e));
  }
  if (size >= IPC_MAX_ALLOCATION)
    return kvr_err::set(KV_EINVAL, "the pointer lies in an allocation of %zu bytes: handles are limited "
                        "to allocations below 2 GiB (export from a smaller allocation)", size);
  const uint64_t off = (uint64_t)(reinterpret_cast<const char*>(ptr) - reinterpret_cast<const char*>(base));
  if (off + bytes > size)
    return kvr_err::set(KV_EINVAL, "%llu bytes at offset %llu exceed the %zu-byte allocation",
                        (unsigned long long)bytes, (unsigned long long)off, size);
  hipIpcMemHandle_t h;
  e = hipIpcGetMemHandle(&h, base);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return kvr_err::set(KV_EDEVICE, "hipIpcGetMemHandle failed: %s", hipGetErrorString(e));
  }
  std::memcpy(out->ipc, &h, sizeof h);
  out->offset = off;
  out->bytes = bytes;
  out->owner_pid = (int64_t)getpid();
  out->device = attr.device;
  return kvr_err::clear();
}

kv_status kv_ipc_owner_alive(const kv_ipc_handle* h) {
  if (!h) return kvr_err::set(KV_EINVAL, "null handle");
  if (h->owner_pid <= 0) return kvr_err::set(KV_EINVAL, "handle has no owner process id");
  if (kill((pid_t)h->owner_pid, 0) == 0 || errno == EPERM) return kvr_err::clear();
  return kvr_err::set(KV_ESTATE, "owner process %lld is gone", (long long)h->owner_pid);
}

kv_status kv_ipc_open(const kv_ipc_handle* h, void** out) {
  if (!h || !out) return kvr_err::set(KV_EINVAL, "null argument");
  *out = nullptr;
  kv_status st = kv_ipc_owner_alive(h);
  if (st != KV_OK) return st;
  if (h->owner_pid == (int64_t)getpid())
    return kvr_err::set(KV_EINVAL, "the owner cannot open its own handle");
  int prev = 0;
  if (hipGetDevice(&prev) != hipSuccess || hipSetDevice(h->device) != hipSuccess) {
    (void)hipGetLastError();
    return kvr_err::set(KV_EDEVICE, "cannot select device %d", h->device);
  }
  hipIpcMemHandle_t ih;
  std::memcpy(&ih, h->ipc, sizeof ih);
  void* base = nullptr;
  hipError_t e = hipIpcOpenMemHandle(&base, ih, hipIpcMemLazyEnablePeerAccess);
  (void)hipSetDevice(prev);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return kvr_err::set(KV_EDEVICE, "hipIpcOpenMemHandle failed: %s", hipGetErrorString(e));
  }
  void* p = reinterpret_cast<char*>(base) + h->offset;
  {
    std::lock_guard<std::mutex> g(g_mu);
    g_opened[p] = base;
  }
  *out = p;
  return kvr_err::clear();
}

kv_status kv_ipc_close(void* ptr) {
  void* base = nullptr;
  {
    std::lock_guard<std::mutex> g(g_mu);
    auto it = g_opened.find(ptr);
    if (it == g_opened.end()) return kvr_err::set(KV_ESTATE, "pointer was not opened by kv_ipc_open");
    base = it->second;
    g_opened.erase(it);
  }
  const hipError_t e = hipIpcCloseMemHandle(base);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return kvr_err::set(KV_EDEVICE, "hipIpcCloseMemHandle failed: %s", hipGetErrorString(e));
  }
  return kvr_err::clear();
}

}  // extern "C"
