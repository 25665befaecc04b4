// Host side of the C ABI declared in include/vc_jointattn.h: argument
// validation, workspace layout, device check and kernel launches. Nothing
// here allocates, frees or synchronises.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <limits>
#include <mutex>

#include "common.hpp"
#include "vc_jointattn.h"

namespace {

constexpr int kMaxDevices = 64;

struct DeviceInfo {
  std::once_flag once;
  bool is_gfx950 = false;
  int cus = 0;  // compute units
};
DeviceInfo g_devices[kMaxDevices];

vc_status check_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return VC_ERR_DEVICE;
  DeviceInfo& di = g_devices[dev];
  std::call_once(di.once, [&] {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) == hipSuccess) {
      di.is_gfx950 = strncmp(prop.gcnArchName, "gfx950", 6) == 0;
      di.cus = prop.multiProcessorCount;
    }
  });
  return di.is_gfx950 ? VC_OK : VC_ERR_DEVICE;
}

// Workspace of vc_jointattn_fwd_noalloc: a file-scope device array (each device holds its
// own copy from the library's first use on it until the process ends). In host code
// `scratch` names a host-side stand-in, not device memory: kernels and copies take the
// device address looked up below, never the array's name.
static __device__ __align__(256) char scratch[VC_JOINTATTN_NOALLOC_SCRATCH_BYTES];

struct ScratchAddr {
  std::once_flag once;
  void* ptr = nullptr;
};
ScratchAddr g_scratch[kMaxDevices];

// Device address of this device's copy of `scratch`, looked up once per device with that
// device current (the caller has checked it with check_device); NULL if the lookup failed.
void* scratch_ptr() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  ScratchAddr& sa = g_scratch[dev];
  std::call_once(sa.once, [&] {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) == hipSuccess) sa.ptr = p;
  });
  return sa.ptr;
}

// Compute units of the current device (after check_device succeeded).
int device_cus() {
  int dev = 0;
  (void)hipGetDevice(&dev);
  return g_devices[dev].cus;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

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

int ntiles(int64_t n) { return (int)((n + vcja::kTileTok - 1) / vcja::kTileTok); }

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Transposed token tiles of one [B, N, H, D] tensor.
size_t tiles_bytes(const vc_jointattn_desc* d, int64_t n) {
  return align256((size_t)d->batch * d->heads * ntiles(n) * vcja::tile_elems(d->head_dim) * sizeof(__bf16));
}

// Per-row fp32 array [B, H, Npad].
size_t rows_bytes(const vc_jointattn_desc* d, int64_t n) {
  return align256((size_t)d->batch * d->heads * (size_t)ntiles(n) * vcja::kTileTok * sizeof(float));
}

// Joint attention: split of the last, partial round of a kernel's dispatch. With W items
// (256-row blocks x heads x samples) on `cus` compute units, the R = W mod cus items of the
// last round are each split into C = cus / R workgroups over runs of `span` tiles along the
// other token axis, so that the round ends after about 1/C of an item's time. At most
// kTailMaxWgs split workgroups (the workspace is planned for that many).
constexpr int kTailMaxWgs = 256;
constexpr int kRowsPerItem = 256;
struct TailPlan {
  int items, chunks, span;
};
TailPlan tail_plan(int64_t work_items, int ntile, int cus) {
  cus = std::min(cus, kTailMaxWgs);
  if (cus < 2 || work_items <= cus) return TailPlan{0, 1, 0};
  const int r = (int)(work_items % cus);
  if (r == 0 || cus / r < 2) return TailPlan{0, 1, 0};
  const int span = (ntile + cus / r - 1) / (cus / r);
  return TailPlan{r, (ntile + span - 1) / span, span};
}
// Items of the joint kernels (256-row blocks x heads x samples).
int64_t joint_items(const vc_jointattn_desc* d, int64_t n) {
  return ((n + kRowsPerItem - 1) / kRowsPerItem) * d->heads * d->batch;
}
// fp32 partials of the split tail: dK and dV of up to kTailMaxWgs workgroups of 256 keys
// (the dQ pass reuses the region for its single tensor).
size_t tail_part_bytes(const vc_jointattn_desc* d, int64_t n) {
  const int64_t wgs = std::min<int64_t>(kTailMaxWgs, joint_items(d, n));
  return align256((size_t)2 * wgs * kRowsPerItem * d->head_dim * sizeof(float));
}

// Fused backward: the key blocks [0, fused_dq_blocks) add their dQ share with atomics in
// the key-stationary pass; the dQ pass covers the others. Per key block, the atomics (an
// fp32 dQ tile per query tile) cost about what the dQ pass's recomputation of S and dP
// costs at head_dim 128, so the backward's time is nearly flat in the fraction between 1/2
// and 7/8 there; 65% measured fastest on the long workload (ragged-text and max-length
// workloads: within 1% from 65% to 80%). At head_dim 64 fusing every key block is fastest
// (medium workload: 1.85 ms against 2.02 at 65% and 2.11 for the separate passes); the dQ
// pass then only converts the accumulator.
constexpr int kFusedDqPercent128 = 65;
constexpr int kFusedDqPercent64 = 100;
// The fused pass addresses a sample's fp32 dQ accumulator with 32-bit element offsets, so it
// runs only while a sample's N*H*D elements fit in 32 bits; larger inputs take the separate
// passes.
bool dq_offsets_fit(const vc_jointattn_desc* d, int64_t n) {
  return n * d->heads * d->head_dim < ((int64_t)1 << 32);
}
int fused_dq_blocks(const vc_jointattn_desc* d, int64_t n) {
  if (!dq_offsets_fit(d, n)) return 0;
  const int nblk = (int)((n + vcja::kDkdvKeys - 1) / vcja::kDkdvKeys);
  const int pct = d->head_dim == 128 ? kFusedDqPercent128 : kFusedDqPercent64;
  return (int)(((int64_t)nblk * pct + 50) / 100);
}
// Every key block carries its dQ share: no dQ pass over key tiles (and no token-major K).
bool all_keys_fused(const vc_jointattn_desc* d, int64_t n) {
  return (int64_t)fused_dq_blocks(d, n) * vcja::kDkdvKeys >= n;
}

// Forward workspace: V^T tiles | split-tail partials (unnormalised O, base, sum per row).
size_t fwd_tail_bytes(const vc_jointattn_desc* d, int64_t n) {
  const int64_t wgs = std::min<int64_t>(kTailMaxWgs, joint_items(d, n));
  return align256((size_t)wgs * kRowsPerItem * (d->head_dim + 2) * sizeof(float));
}
size_t fwd_ws_bytes(const vc_jointattn_desc* d, int64_t n) { return tiles_bytes(d, n) + fwd_tail_bytes(d, n); }

// Backward workspace: -D | LSE*log2(e) | Q^T tiles | dO^T tiles | K^T tiles | tail partials.
struct BwdWorkspace {
  float* dd;
  float* lse2;
  __bf16* qt;
  __bf16* dot;
  __bf16* kt;
};

size_t bwd_ws_bytes(const vc_jointattn_desc* d, int64_t n) {
  return 2 * rows_bytes(d, n) + 3 * tiles_bytes(d, n) + tail_part_bytes(d, n);
}
float* tail_part_of(const vc_jointattn_desc* d, int64_t n, void* ws) {
  return reinterpret_cast<float*>(static_cast<char*>(ws) + 2 * rows_bytes(d, n) + 3 * tiles_bytes(d, n));
}

BwdWorkspace split_bwd_ws(const vc_jointattn_desc* d, int64_t n, void* ws) {
  char* p = static_cast<char*>(ws);
  const size_t rb = rows_bytes(d, n), tb = tiles_bytes(d, n);
  return BwdWorkspace{reinterpret_cast<float*>(p), reinterpret_cast<float*>(p + rb),
                      reinterpret_cast<__bf16*>(p + 2 * rb), reinterpret_cast<__bf16*>(p + 2 * rb + tb),
                      reinterpret_cast<__bf16*>(p + 2 * rb + 2 * tb)};
}

// Spatial branch: split of the text key blocks' video query tiles into chunks of about one
// frame (at least kMinTextSpan tiles), so that no dK/dV workgroup visits every video tile.
constexpr int kMinTextSpan = 8;
constexpr int kMaxTextChunks = 64;
struct TextSplit {
  int blocks, chunks, span;
};
TextSplit text_split(const vc_jointattn_desc* d, int64_t n) {
  const int T = d->text_slot;
  const int blocks = (T + vcja::kDkdvKeys - 1) / vcja::kDkdvKeys;
  const int nvq = ntiles(n) - T / vcja::kTileTok;  // tiles holding video queries
  const int L = d->grid_h * d->grid_w;
  const int span = std::max((L + vcja::kTileTok - 1) / vcja::kTileTok + 1, kMinTextSpan);
  const int chunks = blocks ? std::min(kMaxTextChunks, (nvq + span - 1) / span) : 1;
  if (chunks < 2) return TextSplit{blocks, 1, nvq};
  return TextSplit{blocks, chunks, (nvq + chunks - 1) / chunks};
}
// fp32 partial dK and dV of the split text blocks.
size_t text_part_bytes(const vc_jointattn_desc* d, int64_t n) {
  const TextSplit t = text_split(d, n);
  if (t.chunks < 2) return 0;
  return align256((size_t)2 * t.chunks * d->batch * d->heads * t.blocks * vcja::kDkdvKeys * d->head_dim *
                  sizeof(float));
}
size_t spatial_bwd_ws_bytes(const vc_jointattn_desc* d, int64_t n) {
  return bwd_ws_bytes(d, n) + text_part_bytes(d, n);
}

vc_status check_ws(void* ws, size_t have, size_t need) {
  if (!ws) return VC_ERR_WORKSPACE;
  if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0) return VC_ERR_ALIGN;
  if (have < need) return VC_ERR_WORKSPACE;
  return VC_OK;
}

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// Temporal branch arguments common to the forward and the backward.
vcja::TemporalArgs temporal_args(const vc_jointattn_desc* d, int64_t n) {
  vcja::TemporalArgs a{};
  a.B = d->batch;
  a.H = d->heads;
  a.N = (int)n;
  a.T = d->text_slot;
  a.F = d->frames;
  a.L = d->grid_h * d->grid_w;
  a.G = d->frames <= vcja::kMaxTemporalFramesShort ? 32 / d->frames : 1;
  a.npad = ntiles(n) * vcja::kTileTok;
  a.scale = d->softmax_scale > 0.0f ? d->softmax_scale : 1.0f / sqrtf((float)d->head_dim);
  a.scale_log2 = a.scale * vcja::kLog2e;
  return a;
}
inline const __bf16* bf(const void* p) { return static_cast<const __bf16*>(p); }

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
    case VC_ERR_ALIAS: return "an output is the same buffer as another output";
    case VC_ERR_SCRATCH:
      return "the problem needs more workspace than the no-allocation entry point's fixed scratch array holds";
    default: return "unknown status";
  }
}

int64_t vc_jointattn_tokens(const vc_jointattn_desc* desc) {
  int64_t n = 0;
  const vc_status st = check_desc(desc, &n);
  return st == VC_OK ? n : (int64_t)st;
}

size_t vc_jointattn_fwd_workspace_bytes(const vc_jointattn_desc* desc) {
  int64_t n = 0;
  if (check_desc(desc, &n) != VC_OK) return 0;
  return fwd_ws_bytes(desc, n);
}

size_t vc_jointattn_bwd_workspace_bytes(const vc_jointattn_desc* desc) {
  int64_t n = 0;
  if (check_desc(desc, &n) != VC_OK) return 0;
  return bwd_ws_bytes(desc, n);
}

int64_t vc_jointattn_fused_dq_keys(const vc_jointattn_desc* desc) {
  int64_t n = 0;
  const vc_status st = check_desc(desc, &n);
  if (st != VC_OK) return (int64_t)st;
  return std::min<int64_t>(n, (int64_t)fused_dq_blocks(desc, n) * vcja::kDkdvKeys);
}

size_t vc_spatialattn_bwd_workspace_bytes(const vc_jointattn_desc* desc) {
  int64_t n = 0;
  if (check_desc(desc, &n) != VC_OK) return 0;
  return spatial_bwd_ws_bytes(desc, n);
}

}  // extern "C"

namespace {

// Token-major copies a backward's stage 1 makes: none (every key's dQ share added in the
// key-stationary pass), of k (read by the dQ pass), or of q, dout and k (the separate passes).
enum class StageTiles { kNone, kKeys, kAll };
vc_status prepare_impl(const vc_jointattn_desc* desc, const void* q, const void* k, const void* o, const float* lse,
                       const void* dout, void* workspace, size_t workspace_bytes, void* stream, StageTiles tiles);

// Joint attention (frame_len 0) or the spatial branch (frame_len = tokens per frame).
vc_status fwd_impl(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v,
                   const int32_t* text_len, const uint8_t* key_mask, void* o, float* lse, void* workspace,
                   size_t workspace_bytes, void* stream, bool spatial) {
  int64_t n = 0;
  vc_status st = check_desc(desc, &n);
  if (st != VC_OK) return st;
  if (!q || !k || !v || !o || !lse) return VC_ERR_NULL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(lse) || !aligned4(text_len))
    return VC_ERR_ALIGN;
  if ((st = check_ws(workspace, workspace_bytes, fwd_ws_bytes(desc, n))) != VC_OK) return st;
  if ((st = check_device()) != VC_OK) return st;
  __bf16* vt = static_cast<__bf16*>(workspace);
  if (vcja::launch_token_tiles(bf(v), vt, desc->batch, desc->heads, (int)n, desc->head_dim, as_stream(stream)) !=
      hipSuccess)
    return VC_ERR_HIP;
  vcja::FwdArgs a;
  a.q = bf(q);
  a.k = bf(k);
  a.vt = vt;
  a.text_len = text_len;
  a.key_mask = key_mask;
  a.o = static_cast<__bf16*>(o);
  a.lse = lse;
  a.B = desc->batch;
  a.H = desc->heads;
  a.N = (int)n;
  a.T = desc->text_slot;
  a.ntile = ntiles(n);
  a.frame_len = spatial ? desc->grid_h * desc->grid_w : 0;
  a.scale_log2 = scale_of(desc) * vcja::kLog2e;
  const TailPlan tp = spatial ? TailPlan{0, 1, 0} : tail_plan(joint_items(desc, n), ntiles(n), device_cus());
  a.tail_part = reinterpret_cast<float*>(static_cast<char*>(workspace) + tiles_bytes(desc, n));
  a.tail_blocks = tp.items;
  a.tail_chunks = tp.chunks;
  a.tail_span = tp.span;
  // Spatial branch: text rows are not queries; their o and lse are written here.
  if (spatial && vcja::launch_text_rows(a.o, nullptr, nullptr, lse, a.B, a.H, a.N, a.T, desc->head_dim,
                                        as_stream(stream)) != hipSuccess)
    return VC_ERR_HIP;
  return vcja::launch_fwd(a, desc->head_dim, as_stream(stream)) == hipSuccess ? VC_OK : VC_ERR_HIP;
}

}  // namespace

extern "C" {

vc_status vc_jointattn_fwd(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v,
                           const int32_t* text_len, const uint8_t* key_mask, void* o, float* lse, void* workspace,
                           size_t workspace_bytes, void* stream) {
  return fwd_impl(desc, q, k, v, text_len, key_mask, o, lse, workspace, workspace_bytes, stream, false);
}

vc_status vc_jointattn_fwd_noalloc(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v,
                                   const int32_t* text_len, const uint8_t* key_mask, void* o, float* lse,
                                   void* stream) {
  int64_t n = 0;
  vc_status st = check_desc(desc, &n);
  if (st != VC_OK) return st;
  if (fwd_ws_bytes(desc, n) > VC_JOINTATTN_NOALLOC_SCRATCH_BYTES) return VC_ERR_SCRATCH;
  if ((st = check_device()) != VC_OK) return st;
  void* ws = scratch_ptr();
  if (!ws) return VC_ERR_HIP;
  return fwd_impl(desc, q, k, v, text_len, key_mask, o, lse, ws, VC_JOINTATTN_NOALLOC_SCRATCH_BYTES, stream,
                  false);
}

vc_status vc_spatialattn_fwd(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v,
                             const int32_t* text_len, const uint8_t* key_mask, void* o, float* lse, void* workspace,
                             size_t workspace_bytes, void* stream) {
  return fwd_impl(desc, q, k, v, text_len, key_mask, o, lse, workspace, workspace_bytes, stream, true);
}

vc_status vc_jointattn_bwd_prepare(const vc_jointattn_desc* desc, const void* q, const void* k, const void* o,
                                   const float* lse, const void* dout, void* workspace, size_t workspace_bytes,
                                   void* stream) {
  int64_t n = 0;
  const vc_status st = check_desc(desc, &n);
  if (st != VC_OK) return st;
  const StageTiles tiles = desc->deterministic     ? StageTiles::kAll
                           : all_keys_fused(desc, n) ? StageTiles::kNone
                                                     : StageTiles::kKeys;
  return prepare_impl(desc, q, k, o, lse, dout, workspace, workspace_bytes, stream, tiles);
}

}  // extern "C"

namespace {

// Backward stage 1 and the token-major copies `tiles` asks for: those of q and dout are read
// by the separate dK/dV pass only, that of k by a dQ pass over key tiles.
vc_status prepare_impl(const vc_jointattn_desc* desc, const void* q, const void* k, const void* o, const float* lse,
                       const void* dout, void* workspace, size_t workspace_bytes, void* stream, StageTiles tiles) {
  int64_t n = 0;
  vc_status st = check_desc(desc, &n);
  if (st != VC_OK) return st;
  if (!q || !k || !o || !lse || !dout) return VC_ERR_NULL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(o) || !aligned16(lse) || !aligned16(dout)) return VC_ERR_ALIGN;
  if ((st = check_ws(workspace, workspace_bytes, bwd_ws_bytes(desc, n))) != VC_OK) return st;
  if ((st = check_device()) != VC_OK) return st;
  const BwdWorkspace w = split_bwd_ws(desc, n, workspace);
  const int B = desc->batch, H = desc->heads, D = desc->head_dim, N = (int)n;
  hipStream_t s = as_stream(stream);
  if (vcja::launch_bwd_prepare(bf(o), lse, bf(dout), w.dd, w.lse2, B, H, N, ntiles(n) * vcja::kTileTok, D, s) !=
      hipSuccess)
    return VC_ERR_HIP;
  if (tiles == StageTiles::kAll && (vcja::launch_token_tiles(bf(q), w.qt, B, H, N, D, s) != hipSuccess ||
                                    vcja::launch_token_tiles(bf(dout), w.dot, B, H, N, D, s) != hipSuccess))
    return VC_ERR_HIP;
  if (tiles != StageTiles::kNone && vcja::launch_token_tiles(bf(k), w.kt, B, H, N, D, s) != hipSuccess)
    return VC_ERR_HIP;
  return VC_OK;
}

vc_status dkdv_impl(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v, const void* dout,
                    const int32_t* text_len, const uint8_t* key_mask, void* dk, void* dv, void* workspace,
                    size_t workspace_bytes, void* stream, bool spatial, bool fused = false,
                    bool staged = false) {
  int64_t n = 0;
  vc_status st = check_desc(desc, &n);
  if (st != VC_OK) return st;
  if (!q || !k || !v || !dout || !dk || !dv) return VC_ERR_NULL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(dout) || !aligned16(dk) || !aligned16(dv) ||
      !aligned4(text_len))
    return VC_ERR_ALIGN;
  if ((st = check_ws(workspace, workspace_bytes, spatial ? spatial_bwd_ws_bytes(desc, n) : bwd_ws_bytes(desc, n))) !=
      VC_OK)
    return st;
  if ((st = check_device()) != VC_OK) return st;
  // The separate stages 2 and 3 read the token-major copies, which stage 1 makes only for
  // the deterministic backward.
  if (staged && !desc->deterministic) return VC_ERR_UNSUPPORTED;
  const BwdWorkspace w = split_bwd_ws(desc, n, workspace);
  vcja::DkdvArgs a{};
  const TextSplit ts = spatial ? text_split(desc, n) : TextSplit{0, 1, 0};
  a.text_part = reinterpret_cast<float*>(static_cast<char*>(workspace) + bwd_ws_bytes(desc, n));
  a.text_blocks = ts.blocks;
  a.text_chunks = ts.chunks;
  a.text_span = ts.span;
  const TailPlan tp = spatial ? TailPlan{0, 1, 0} : tail_plan(joint_items(desc, n), ntiles(n), device_cus());
  a.tail_part = tail_part_of(desc, n, workspace);
  a.tail_blocks = tp.items;
  a.tail_chunks = tp.chunks;
  a.tail_span = tp.span;
  a.q = bf(q);
  a.k = bf(k);
  a.v = bf(v);
  a.dout = bf(dout);
  a.qt = w.qt;
  a.dot = w.dot;
  a.lse2 = w.lse2;
  a.dd = w.dd;
  a.text_len = text_len;
  a.key_mask = key_mask;
  a.dk = static_cast<__bf16*>(dk);
  a.dv = static_cast<__bf16*>(dv);
  // Fused dQ: the fp32 accumulator takes the place of the transposed Q and dO tiles, which
  // the fused backward does not make (2 tile sets >= 4 bytes per element of dq).
  a.dq_acc = fused ? reinterpret_cast<float*>(w.qt) : nullptr;
  a.dq_blocks = !fused ? 0 : spatial ? std::numeric_limits<int>::max() : fused_dq_blocks(desc, n);
  a.B = desc->batch;
  a.H = desc->heads;
  a.N = (int)n;
  a.T = desc->text_slot;
  a.ntile = ntiles(n);
  a.frame_len = spatial ? desc->grid_h * desc->grid_w : 0;
  a.scale = scale_of(desc);
  a.scale_log2 = a.scale * vcja::kLog2e;
  return vcja::launch_bwd_dkdv(a, desc->head_dim, as_stream(stream)) == hipSuccess ? VC_OK : VC_ERR_HIP;
}

vc_status dq_impl(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v, const void* dout,
                  const int32_t* text_len, const uint8_t* key_mask, void* dq, void* workspace,
                  size_t workspace_bytes, void* stream, bool spatial, bool fused = false) {
  int64_t n = 0;
  vc_status st = check_desc(desc, &n);
  if (st != VC_OK) return st;
  if (!q || !k || !v || !dout || !dq) return VC_ERR_NULL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(dout) || !aligned16(dq) || !aligned4(text_len))
    return VC_ERR_ALIGN;
  if ((st = check_ws(workspace, workspace_bytes, bwd_ws_bytes(desc, n))) != VC_OK) return st;
  if ((st = check_device()) != VC_OK) return st;
  const BwdWorkspace w = split_bwd_ws(desc, n, workspace);
  vcja::DqArgs a{};
  // Completing a fused backward: the key tiles of the blocks that did not add their dQ
  // share, plus the accumulator the others filled; when every block added its share, the
  // accumulator alone, scaled and rounded.
  if (fused) {
    if (spatial || all_keys_fused(desc, n)) {
      hipStream_t s = as_stream(stream);
      if (vcja::launch_dq_from_acc(reinterpret_cast<const float*>(w.qt), static_cast<__bf16*>(dq),
                                   (size_t)desc->batch * n * desc->heads * desc->head_dim, scale_of(desc),
                                   s) != hipSuccess)
        return VC_ERR_HIP;
      // Spatial branch: text rows are not queries; their dq is zero.
      if (spatial && vcja::launch_text_rows(static_cast<__bf16*>(dq), nullptr, nullptr, nullptr, desc->batch,
                                            desc->heads, (int)n, desc->text_slot, desc->head_dim, s) != hipSuccess)
        return VC_ERR_HIP;
      return VC_OK;
    }
    a.kt_min = fused_dq_blocks(desc, n) * (vcja::kDkdvKeys / vcja::kTileTok);
    a.dq_acc = reinterpret_cast<const float*>(w.qt);
  }
  a.q = bf(q);
  a.k = bf(k);
  a.v = bf(v);
  a.dout = bf(dout);
  a.kt = w.kt;
  a.lse2 = w.lse2;
  a.dd = w.dd;
  a.text_len = text_len;
  a.key_mask = key_mask;
  a.dq = static_cast<__bf16*>(dq);
  const TailPlan tp = spatial ? TailPlan{0, 1, 0} : tail_plan(joint_items(desc, n), ntiles(n), device_cus());
  a.tail_part = tail_part_of(desc, n, workspace);
  a.tail_blocks = tp.items;
  a.tail_chunks = tp.chunks;
  a.tail_span = tp.span;
  a.B = desc->batch;
  a.H = desc->heads;
  a.N = (int)n;
  a.T = desc->text_slot;
  a.ntile = ntiles(n);
  a.frame_len = spatial ? desc->grid_h * desc->grid_w : 0;
  a.scale = scale_of(desc);
  a.scale_log2 = a.scale * vcja::kLog2e;
  // Spatial branch: text rows are not queries; their dq is zero.
  if (spatial && vcja::launch_text_rows(a.dq, nullptr, nullptr, nullptr, a.B, a.H, a.N, a.T, desc->head_dim,
                                        as_stream(stream)) != hipSuccess)
    return VC_ERR_HIP;
  return vcja::launch_bwd_dq(a, desc->head_dim, as_stream(stream)) == hipSuccess ? VC_OK : VC_ERR_HIP;
}

vc_status bwd_impl(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v, const void* o,
                   const float* lse, const void* dout, const int32_t* text_len, const uint8_t* key_mask, void* dq,
                   void* dk, void* dv, void* workspace, size_t workspace_bytes, void* stream, bool spatial) {
  int64_t n = 0;
  vc_status st = check_desc(desc, &n);
  if (st != VC_OK) return st;
  if (!q || !k || !v || !o || !lse || !dout || !dq || !dk || !dv) return VC_ERR_NULL;
  if (spatial && (st = check_ws(workspace, workspace_bytes, spatial_bwd_ws_bytes(desc, n))) != VC_OK) return st;
  // dQ fused into the key-stationary kernel (atomics) unless the caller asks for bitwise
  // reproducible results: joint attention for its leading key blocks (the dQ pass covers
  // the others), the spatial branch for every key block (a video query row gets the shares
  // of 16 key blocks at 720p, so the atomics are few); neither past 32-bit dQ offsets.
  if (!desc->deterministic && (spatial ? dq_offsets_fit(desc, n) : fused_dq_blocks(desc, n) > 0)) {
    const StageTiles tiles = (spatial || all_keys_fused(desc, n)) ? StageTiles::kNone : StageTiles::kKeys;
    if ((st = prepare_impl(desc, q, k, o, lse, dout, workspace, workspace_bytes, stream, tiles)) != VC_OK ||
        (st = dkdv_impl(desc, q, k, v, dout, text_len, key_mask, dk, dv, workspace, workspace_bytes, stream,
                        spatial, true)) != VC_OK)
      return st;
    return dq_impl(desc, q, k, v, dout, text_len, key_mask, dq, workspace, workspace_bytes, stream, spatial, true);
  }
  if ((st = prepare_impl(desc, q, k, o, lse, dout, workspace, workspace_bytes, stream, StageTiles::kAll)) != VC_OK)
    return st;
  if ((st = dkdv_impl(desc, q, k, v, dout, text_len, key_mask, dk, dv, workspace, workspace_bytes, stream,
                      spatial)) != VC_OK)
    return st;
  return dq_impl(desc, q, k, v, dout, text_len, key_mask, dq, workspace, workspace_bytes, stream, spatial);
}

}  // namespace

extern "C" {

vc_status vc_jointattn_bwd_dkdv(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v,
                                const void* dout, const int32_t* text_len, const uint8_t* key_mask, void* dk,
                                void* dv, void* workspace, size_t workspace_bytes, void* stream) {
  return dkdv_impl(desc, q, k, v, dout, text_len, key_mask, dk, dv, workspace, workspace_bytes, stream, false,
                   false, true);
}

vc_status vc_jointattn_bwd_dq(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v,
                              const void* dout, const int32_t* text_len, const uint8_t* key_mask, void* dq,
                              void* workspace, size_t workspace_bytes, void* stream) {
  return dq_impl(desc, q, k, v, dout, text_len, key_mask, dq, workspace, workspace_bytes, stream, false,
                 desc && !desc->deterministic);
}

vc_status vc_jointattn_bwd_fused(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v,
                                 const void* dout, const int32_t* text_len, const uint8_t* key_mask, void* dk,
                                 void* dv, void* workspace, size_t workspace_bytes, void* stream) {
  return dkdv_impl(desc, q, k, v, dout, text_len, key_mask, dk, dv, workspace, workspace_bytes, stream, false, true);
}

vc_status vc_jointattn_bwd(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v, const void* o,
                           const float* lse, const void* dout, const int32_t* text_len, const uint8_t* key_mask,
                           void* dq, void* dk, void* dv, void* workspace, size_t workspace_bytes, void* stream) {
  return bwd_impl(desc, q, k, v, o, lse, dout, text_len, key_mask, dq, dk, dv, workspace, workspace_bytes, stream,
                  false);
}

vc_status vc_spatialattn_bwd(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v,
                             const void* o, const float* lse, const void* dout, const int32_t* text_len,
                             const uint8_t* key_mask, void* dq, void* dk, void* dv, void* workspace,
                             size_t workspace_bytes, void* stream) {
  return bwd_impl(desc, q, k, v, o, lse, dout, text_len, key_mask, dq, dk, dv, workspace, workspace_bytes, stream,
                  true);
}

}  // extern "C"

namespace {

// Temporal forward; with `out`, also the branch sum out = o_joint + o_spatial + o.
vc_status temporal_fwd_impl(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v,
                            const uint8_t* key_mask, const void* o_joint, const void* o_spatial, void* o, float* lse,
                            void* out, void* stream) {
  int64_t n = 0;
  vc_status st = check_desc(desc, &n);
  if (st != VC_OK) return st;
  if (desc->frames > vcja::kMaxTemporalFramesLong) return VC_ERR_SHAPE;
  if (!q || !k || !v || !o || !lse) return VC_ERR_NULL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(lse) || !aligned16(o_joint) ||
      !aligned16(o_spatial) || !aligned16(out))
    return VC_ERR_ALIGN;
  if (out && out == o) return VC_ERR_ALIAS;
  if ((st = check_device()) != VC_OK) return st;
  vcja::TemporalArgs a = temporal_args(desc, n);
  a.q = bf(q);
  a.k = bf(k);
  a.v = bf(v);
  a.key_mask = key_mask;
  a.o = static_cast<__bf16*>(o);
  a.lse = lse;
  a.sum_a = bf(o_joint);
  a.sum_b = bf(o_spatial);
  a.sum_out = static_cast<__bf16*>(out);
  hipStream_t s = as_stream(stream);
  if (vcja::launch_text_rows(a.o, nullptr, nullptr, lse, a.B, a.H, a.N, a.T, desc->head_dim, s) != hipSuccess)
    return VC_ERR_HIP;
  // text rows of the sum: this branch contributes zero there
  if (out && vcja::launch_branch_sum(a.sum_a, a.sum_b, nullptr, a.sum_out, a.B, a.N, a.T, a.H * desc->head_dim, s) !=
                 hipSuccess)
    return VC_ERR_HIP;
  const hipError_t e = desc->frames > vcja::kMaxTemporalFramesShort
                          ? vcja::launch_temporal_long_fwd(a, desc->head_dim, device_cus(), s)
                          : vcja::launch_temporal_fwd(a, desc->head_dim, s);
  return e == hipSuccess ? VC_OK : VC_ERR_HIP;
}

}  // namespace

extern "C" {

vc_status vc_temporalattn_fwd(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v,
                              const uint8_t* key_mask, void* o, float* lse, void* stream) {
  return temporal_fwd_impl(desc, q, k, v, key_mask, nullptr, nullptr, o, lse, nullptr, stream);
}

vc_status vc_temporalattn_fwd_sum(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v,
                                  const uint8_t* key_mask, const void* o_joint, const void* o_spatial, void* o,
                                  float* lse, void* out, void* stream) {
  if (!out) return VC_ERR_NULL;
  return temporal_fwd_impl(desc, q, k, v, key_mask, o_joint, o_spatial, o, lse, out, stream);
}

vc_status vc_branchsum(const vc_jointattn_desc* desc, const void* o_joint, const void* o_spatial,
                       const void* o_temporal, void* out, void* stream) {
  int64_t n = 0;
  vc_status st = check_desc(desc, &n);
  if (st != VC_OK) return st;
  if (!out || (!o_joint && !o_spatial && !o_temporal)) return VC_ERR_NULL;
  if (!aligned16(o_joint) || !aligned16(o_spatial) || !aligned16(o_temporal) || !aligned16(out)) return VC_ERR_ALIGN;
  if ((st = check_device()) != VC_OK) return st;
  const int rows = (int)n;
  return vcja::launch_branch_sum(bf(o_joint), bf(o_spatial), bf(o_temporal), static_cast<__bf16*>(out),
                                 desc->batch, rows, rows, desc->heads * desc->head_dim, as_stream(stream)) == hipSuccess
             ? VC_OK
             : VC_ERR_HIP;
}

size_t vc_temporalattn_bwd_workspace_bytes(const vc_jointattn_desc* desc) {
  int64_t n = 0;
  if (check_desc(desc, &n) != VC_OK) return 0;
  return 2 * rows_bytes(desc, n);
}

vc_status vc_temporalattn_bwd(const vc_jointattn_desc* desc, const void* q, const void* k, const void* v,
                              const void* o, const float* lse, const void* dout, const uint8_t* key_mask, void* dq,
                              void* dk, void* dv, void* /*workspace*/, size_t /*workspace_bytes*/,
                              void* stream) {
  int64_t n = 0;
  vc_status st = check_desc(desc, &n);
  if (st != VC_OK) return st;
  if (desc->frames > vcja::kMaxTemporalFramesLong) return VC_ERR_SHAPE;
  if (!q || !k || !v || !o || !lse || !dout || !dq || !dk || !dv) return VC_ERR_NULL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(lse) || !aligned16(dout) ||
      !aligned16(dq) || !aligned16(dk) || !aligned16(dv))
    return VC_ERR_ALIGN;
  const bool long_clip = desc->frames > vcja::kMaxTemporalFramesShort;
  if ((st = check_device()) != VC_OK) return st;
  vcja::TemporalArgs a = temporal_args(desc, n);
  a.q = bf(q);
  a.k = bf(k);
  a.v = bf(v);
  a.dout = bf(dout);
  a.key_mask = key_mask;
  a.o = static_cast<__bf16*>(dq);
  a.dk = static_cast<__bf16*>(dk);
  a.dv = static_cast<__bf16*>(dv);
  hipStream_t s = as_stream(stream);
  if (vcja::launch_text_rows(a.o, a.dk, a.dv, nullptr, a.B, a.H, a.N, a.T, desc->head_dim, s) != hipSuccess)
    return VC_ERR_HIP;
  // -D and LSE*log2(e) are formed inside the kernels from o and lse: no workspace.
  a.lse = const_cast<float*>(lse);
  a.o_in = bf(o);
  if (long_clip)
    return vcja::launch_temporal_long_bwd(a, desc->head_dim, device_cus(), s) == hipSuccess ? VC_OK : VC_ERR_HIP;
  return vcja::launch_temporal_bwd(a, desc->head_dim, s) == hipSuccess ? VC_OK : VC_ERR_HIP;
}

}  // extern "C"
