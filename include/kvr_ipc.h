/*
 * kvr_ipc.h -- retained state owned by another process.
 *
 * In the paper the weights and the raw KV arena survive a worker failure
 * because independent owner processes hold them (Sec. 4.1, state-isolation
 * paragraph); the replacement worker obtains them as pointers and metadata
 * (Sec. 6, shadow-worker integration), checks that the owners are alive and
 * the GPU healthy before reusing anything (Sec. 4.2 Handover, steps 1-2) and
 * refuses reuse otherwise.  These calls carry a device allocation across
 * processes on one GPU with HIP IPC memory handles, tagged with the owner's
 * process id so the importer can check the owner before opening it.  The
 * importer then binds the opened arena with kv_arena_bind (which runs the
 * GPU health probe) and passes opened weight pointers in kv_weights.
 * Same conventions as kvr.h.
 */
#ifndef KVR_IPC_H
#define KVR_IPC_H

#include <stdint.h>

#include "kvr.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Plain bytes, safe to copy through a pipe or file. */
typedef struct {
  uint8_t ipc[64];    /* the HIP IPC memory handle of the whole allocation     */
  uint64_t offset;    /* byte offset of the exported pointer in that allocation */
  uint64_t bytes;     /* bytes the exporter vouches for from that pointer      */
  int64_t owner_pid;  /* process id of the exporter (the owner)                */
  int32_t device;     /* device ordinal the allocation lives on                */
  int32_t reserved;
} kv_ipc_handle;

/* Owner side: describe `bytes` bytes of device memory starting at `ptr` (any
 * pointer inside a device allocation of the calling process, with ptr+bytes
 * inside the same allocation).  A handle covers the whole allocation, and
 * handles are limited to allocations below 2 GiB: larger ones are refused with
 * KV_EINVAL (owners hold large weights and arenas as several allocations of
 * less than 2 GiB each).  KV_EINVAL for null arguments, KV_EDEVICE when HIP
 * does not know the pointer or cannot create a handle. */
kv_status kv_ipc_export(const void* ptr, uint64_t bytes, kv_ipc_handle* out);

/* Importer side: KV_OK when the process owner_pid exists, KV_ESTATE when it
 * has exited (no device access). */
kv_status kv_ipc_owner_alive(const kv_ipc_handle* h);

/* Importer side: check the owner is alive (KV_ESTATE otherwise), then open
 * the handle on h->device and return the exported pointer (the allocation
 * base plus h->offset) in *out.  KV_EINVAL when called by the owner itself,
 * KV_EDEVICE when HIP cannot open the handle.  The mapping stays valid until
 * kv_ipc_close; the owner must keep the allocation alive meanwhile. */
kv_status kv_ipc_open(const kv_ipc_handle* h, void** out);

/* Importer side: unmap a pointer returned by kv_ipc_open. */
kv_status kv_ipc_close(void* ptr);

#ifdef __cplusplus
}
#endif
#endif
