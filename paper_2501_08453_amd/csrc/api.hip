// Host side of the C ABI declared in include/vc_jointattn.h: argument
// validation, workspace layout, device check and kernel launches. Nothing
// here allocates, frees or synchronises.
#include <math.h>
#include <string.h>

#include <mutex>

#include "../../include/vc_jointattn.h"
#include "common.hpp"

namespace {

constexpr int kMaxDevices = 64;

struct DeviceInfo {
  std::once_flag once;
  bool is_gfx950 = false;
};
DeviceInfo g_devices[kMaxDevices];

vc_status check_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return VC_ERR_DEVICE;
  DeviceInfo& di = g_devices[dev];
  std::call_once(di.once, [&] {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) == hipSuccess)
      di.is_gfx950 = strncmp(prop.gcnArchName, "gfx950", 6) == 0;
  });
  return di.is_gfx950 ? VC_OK : VC_ERR_DEVICE;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Validates a descriptor; on success fills N.
vc_status check_desc(const vc_jointattn_desc* d, int64_t* n_out) {
  if (!d) return VC_ERR_NULL;
  if (d->head_dim != 64 && d->head_dim != 128) return VC_ERR_HEAD_DIM;
  if (d->batch < 1 || d->heads < 1 || d->text_slot < 0 || d->frames < 1 || d->grid_h < 1 || d->grid_w < 1)
    return VC_ERR_SHAPE;
  if (d->heads > 65535 || d->batch > 65535) return VC_ERR_SHAPE;
  if (!(d->softmax_scale <= 0.0f || isfinite(d->softmax_scale))) return VC_ERR_SHAPE;
  if (d->deterministic != 0 && d->deterministic != 1) return VC_ERR_SHAPE;
  const int64_t video = (int64_t)d->frames * d->grid_h * d->grid_w;
  const int64_t n = (int64_t)d->text_slot + video;
  if (video <= 0 || n > (int64_t)1 << 30) return VC_ERR_SHAPE;
  // Element counts of a [B, N, H, D] tensor must stay well inside 64-bit byte offsets.
  const int64_t elems = (int64_t)d->batch * n * d->heads * d->head_dim;
  if (elems <= 0 || elems > ((int64_t)1 << 40)) return VC_ERR_SHAPE;
  *n_out = n;
  return VC_OK;
}

float scale_of(const vc_jointattn_desc* d) {
  return d->softmax_scale > 0.0f ? d->softmax_scale : 1.0f / sqrtf((float)d->head_dim);
}

size_t dd_bytes(const vc_jointattn_desc* d, int64_t n) {
  const size_t raw = (size_t)d->batch * d->heads * (size_t)n * sizeof(float);
  return (raw + 255) & ~(size_t)255;
}

size_t ws_bytes(const vc_jointattn_desc* d, int64_t n) {
  return dd_bytes(d, n) + (size_t)d->batch * (size_t)n * d->heads * d->head_dim * sizeof(float);
}

vc_status check_ws(const vc_jointattn_desc* d, int64_t n, void* ws, size_t bytes) {
  if (!ws) return VC_ERR_WORKSPACE;
  if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0) return VC_ERR_ALIGN;
  if (bytes < ws_bytes(d, n)) return VC_ERR_WORKSPACE;
  return VC_OK;
}

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

}  // namespace

extern "C" {

int vc_jointattn_abi_version(void) { return VC_JOINTATTN_ABI_VERSION; }

const char* vc_status_string(int status) {
  switch (status) {
    case VC_OK: return "ok";
    case VC_ERR_NULL: return "a required pointer is NULL";
    case VC_ERR_SHAPE: return "a size is out of range";
    case VC_ERR_HEAD_DIM: return "head_dim must be 64 or 128";
    case VC_ERR_ALIGN: return "a pointer is not sufficiently aligned";
    case VC_ERR_WORKSPACE: return "workspace missing or too small";
    case VC_ERR_DEVICE: return "no current HIP device, or it is not gfx950";
    case VC_ERR_HIP: return "a HIP kernel launch failed";
    case VC_ERR_UNSUPPORTED: return "requested mode is not available";
    default: return "unknown status";
  }
}

int64_t vc_jointattn_tokens(const vc_jointattn_desc* desc) {
  int64_t n = 0;
  const vc_status st = check_desc(desc, &n);
  return st == VC_OK ? n : (int64_t)st;
}

size_t vc_jointattn_bwd_workspace_bytes(const vc_jointattn_desc* desc) {
  int64_t n = 0;
  if (check_desc(desc, &n) != VC_OK) return 0;
  return ws_bytes(desc, n);
}

vc_status vc_jointattn_fwd(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v,
                           const int32_t* text_len, const uint8_t* key_mask, void* o, float* lse, void* stream) {
  int64_t n = 0;
  vc_status st = check_desc(desc, &n);
  if (st != VC_OK) return st;
  if (!q || !k || !v || !o || !lse) return VC_ERR_NULL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(lse)) return VC_ERR_ALIGN;
  if ((reinterpret_cast<uintptr_t>(text_len) & 3u) != 0) return VC_ERR_ALIGN;
  if ((st = check_device()) != VC_OK) return st;
  vcja::FwdArgs a;
  a.q = static_cast<const __bf16*>(q);
  a.k = static_cast<const __bf16*>(k);
  a.v = static_cast<const __bf16*>(v);
  a.text_len = text_len;
  a.key_mask = key_mask;
  a.o = static_cast<__bf16*>(o);
  a.lse = lse;
  a.B = desc->batch;
  a.H = desc->heads;
  a.N = (int)n;
  a.T = desc->text_slot;
  a.scale_log2 = scale_of(desc) * vcja::kLog2e;
  return vcja::launch_fwd(a, desc->head_dim, as_stream(stream)) == hipSuccess ? VC_OK : VC_ERR_HIP;
}

vc_status vc_jointattn_bwd_prepare(const vc_jointattn_desc* desc, const void* o, const void* dout, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  int64_t n = 0;
  vc_status st = check_desc(desc, &n);
  if (st != VC_OK) return st;
  if (!o || !dout) return VC_ERR_NULL;
  if (!aligned16(o) || !aligned16(dout)) return VC_ERR_ALIGN;
  if ((st = check_ws(desc, n, workspace, workspace_bytes)) != VC_OK) return st;
  if ((st = check_device()) != VC_OK) return st;
  float* dd = static_cast<float*>(workspace);
  float* acc = reinterpret_cast<float*>(static_cast<char*>(workspace) + dd_bytes(desc, n));
  const hipError_t e = vcja::launch_bwd_prepare(static_cast<const __bf16*>(o), static_cast<const __bf16*>(dout), dd,
                                                acc, desc->batch, desc->heads, (int)n, desc->head_dim,
                                                as_stream(stream));
  return e == hipSuccess ? VC_OK : VC_ERR_HIP;
}

vc_status vc_jointattn_bwd_main(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v,
                                const float* lse, const void* dout, const int32_t* text_len,
                                const uint8_t* key_mask, void* dk, void* dv, void* workspace,
                                size_t workspace_bytes, void* stream) {
  int64_t n = 0;
  vc_status st = check_desc(desc, &n);
  if (st != VC_OK) return st;
  if (!q || !k || !v || !lse || !dout || !dk || !dv) return VC_ERR_NULL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(lse) || !aligned16(dout) || !aligned16(dk) ||
      !aligned16(dv))
    return VC_ERR_ALIGN;
  if ((reinterpret_cast<uintptr_t>(text_len) & 3u) != 0) return VC_ERR_ALIGN;
  if ((st = check_ws(desc, n, workspace, workspace_bytes)) != VC_OK) return st;
  if (desc->deterministic) return VC_ERR_UNSUPPORTED;
  if ((st = check_device()) != VC_OK) return st;
  vcja::BwdArgs a;
  a.q = static_cast<const __bf16*>(q);
  a.k = static_cast<const __bf16*>(k);
  a.v = static_cast<const __bf16*>(v);
  a.dout = static_cast<const __bf16*>(dout);
  a.lse = lse;
  a.dd = static_cast<const float*>(workspace);
  a.text_len = text_len;
  a.key_mask = key_mask;
  a.dk = static_cast<__bf16*>(dk);
  a.dv = static_cast<__bf16*>(dv);
  a.dq_acc = reinterpret_cast<float*>(static_cast<char*>(workspace) + dd_bytes(desc, n));
  a.B = desc->batch;
  a.H = desc->heads;
  a.N = (int)n;
  a.T = desc->text_slot;
  a.scale = scale_of(desc);
  a.scale_log2 = a.scale * vcja::kLog2e;
  return vcja::launch_bwd_main(a, desc->head_dim, as_stream(stream)) == hipSuccess ? VC_OK : VC_ERR_HIP;
}

vc_status vc_jointattn_bwd_finish(const vc_jointattn_desc* desc, void* dq, void* workspace, size_t workspace_bytes,
                                  void* stream) {
  int64_t n = 0;
  vc_status st = check_desc(desc, &n);
  if (st != VC_OK) return st;
  if (!dq) return VC_ERR_NULL;
  if (!aligned16(dq)) return VC_ERR_ALIGN;
  if ((st = check_ws(desc, n, workspace, workspace_bytes)) != VC_OK) return st;
  if ((st = check_device()) != VC_OK) return st;
  const float* acc = reinterpret_cast<const float*>(static_cast<const char*>(workspace) + dd_bytes(desc, n));
  const hipError_t e =
      vcja::launch_bwd_finish(acc, static_cast<__bf16*>(dq), desc->batch, desc->heads, (int)n, desc->head_dim,
                              as_stream(stream));
  return e == hipSuccess ? VC_OK : VC_ERR_HIP;
}

vc_status vc_jointattn_bwd(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v, const void* o,
                           const float* lse, const void* dout, const int32_t* text_len, const uint8_t* key_mask,
                           void* dq, void* dk, void* dv, void* workspace, size_t workspace_bytes, void* stream) {
  int64_t n = 0;
  vc_status st = check_desc(desc, &n);
  if (st != VC_OK) return st;
  if (!q || !k || !v || !o || !lse || !dout || !dq || !dk || !dv) return VC_ERR_NULL;
  if (desc->deterministic) return VC_ERR_UNSUPPORTED;
  if ((st = vc_jointattn_bwd_prepare(desc, o, dout, workspace, workspace_bytes, stream)) != VC_OK) return st;
  if ((st = vc_jointattn_bwd_main(desc, q, k, v, lse, dout, text_len, key_mask, dk, dv, workspace, workspace_bytes,
                                  stream)) != VC_OK)
    return st;
  return vc_jointattn_bwd_finish(desc, dq, workspace, workspace_bytes, stream);
}

}  // extern "C"
