// Activation offload engine: asynchronous copies of saved activations between device
// memory and pinned host memory, on a copy stream of the engine's own, so that the
// transfers overlap the attention kernels on the caller's stream. Activation offloading
// with stream-overlapped swapping is the paper's single-device complement to
// recomputation (Sec. V-B; measured against recomputation in Sec. VI-D).
//
// Ordering: each copy waits (through an event) for all work the caller's stream has
// queued before the call, so a tensor written by a kernel on that stream can be stored
// right after the launch. vc_offload_wait makes the caller's stream wait for every copy
// issued so far; a stored device buffer must not be overwritten, and a loaded one not
// read, on the caller's stream before that wait. No call blocks the host except
// vc_offload_destroy, which drains the copy stream.
#include <hip/hip_runtime.h>

#include <new>

#include "vc_jointattn.h"

struct vc_offload {
  int device;
  hipStream_t copy;          // copy stream, default priority
  hipEvent_t after_caller;   // recorded on the caller's stream before each copy
  hipEvent_t copies_done;    // recorded on the copy stream by vc_offload_wait
};

namespace {

// Memory type and allocation bounds of p; false if HIP does not know the pointer.
bool query(const void* p, hipMemoryType* type, int* device, char** base, size_t* size) {
  hipPointerAttribute_t attr;
  if (hipPointerGetAttributes(&attr, p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  *type = attr.type;
  *device = attr.device;
  hipDeviceptr_t b = nullptr;
  if (hipMemGetAddressRange(&b, size, const_cast<void*>(p)) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  *base = static_cast<char*>(b);
  return true;
}

// [p, p + bytes) lies in one allocation of the given kind (device memory of `dev`, or
// pinned host memory). Pageable host memory is refused: a copy from it is staged
// synchronously and would not overlap anything.
bool in_allocation(const void* p, size_t bytes, bool host, int dev) {
  hipMemoryType type;
  int owner = -1;
  char* base = nullptr;
  size_t size = 0;
  if (!query(p, &type, &owner, &base, &size)) return false;
  if (host ? type != hipMemoryTypeHost : (type != hipMemoryTypeDevice || owner != dev)) return false;
  const char* c = static_cast<const char*>(p);
  return c >= base && bytes <= size && (size_t)(c - base) <= size - bytes;
}

vc_status issue(vc_offload* h, void* dst, const void* src, size_t bytes, bool to_host, void* stream) {
  if (!h || !dst || !src) return VC_ERR_NULL;
  if (bytes == 0) return VC_OK;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != h->device) return VC_ERR_DEVICE;
  if (!in_allocation(to_host ? dst : src, bytes, true, dev) || !in_allocation(to_host ? src : dst, bytes, false, dev))
    return VC_ERR_UNSUPPORTED;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (hipEventRecord(h->after_caller, s) != hipSuccess || hipStreamWaitEvent(h->copy, h->after_caller, 0) != hipSuccess ||
      hipMemcpyAsync(dst, src, bytes, to_host ? hipMemcpyDeviceToHost : hipMemcpyHostToDevice, h->copy) != hipSuccess)
    return VC_ERR_HIP;
  return VC_OK;
}

void release(vc_offload* h) {
  if (h->copy) {
    (void)hipStreamSynchronize(h->copy);
    (void)hipStreamDestroy(h->copy);
  }
  if (h->after_caller) (void)hipEventDestroy(h->after_caller);
  if (h->copies_done) (void)hipEventDestroy(h->copies_done);
  delete h;
}

}  // namespace

extern "C" {

vc_status vc_offload_create(vc_offload** out) {
  if (!out) return VC_ERR_NULL;
  *out = nullptr;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
    (void)hipGetLastError();
    return VC_ERR_DEVICE;
  }
  vc_offload* h = new (std::nothrow) vc_offload{dev, nullptr, nullptr, nullptr};
  if (!h) return VC_ERR_HIP;
  if (hipStreamCreateWithFlags(&h->copy, hipStreamNonBlocking) != hipSuccess ||
      hipEventCreateWithFlags(&h->after_caller, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&h->copies_done, hipEventDisableTiming) != hipSuccess) {
    release(h);
    return VC_ERR_HIP;
  }
  *out = h;
  return VC_OK;
}

vc_status vc_offload_destroy(vc_offload* h) {
  if (!h) return VC_ERR_NULL;
  release(h);
  return VC_OK;
}

vc_status vc_offload_store(vc_offload* h, void* host_dst, const void* dev_src, size_t bytes, void* stream) {
  return issue(h, host_dst, dev_src, bytes, true, stream);
}

vc_status vc_offload_load(vc_offload* h, void* dev_dst, const void* host_src, size_t bytes, void* stream) {
  return issue(h, dev_dst, host_src, bytes, false, stream);
}

vc_status vc_offload_wait(vc_offload* h, void* stream) {
  if (!h) return VC_ERR_NULL;
  if (hipEventRecord(h->copies_done, h->copy) != hipSuccess ||
      hipStreamWaitEvent(reinterpret_cast<hipStream_t>(stream), h->copies_done, 0) != hipSuccess)
    return VC_ERR_HIP;
  return VC_OK;
}

}  // extern "C"
