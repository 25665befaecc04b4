/*
 * vc_jointattn.h -- C ABI of the joint text-video attention library (gfx950).
 *
 * The operation is the full-sequence branch of the multimodal diffusion block
 * of Vchitect-2.0 (Sec. III-B, "Parallel Transformer Architecture", and the
 * method-overview figure): multi-head self-attention across the concatenation
 * of text tokens and spatio-temporal video tokens (Sec. V-A, "3D and
 * multi-modal nature": attention runs over the concatenated visual and text
 * sequence while other operators treat the two separately). Q, K and V arrive
 * already projected per modality. The paper gives no formula; the library
 * computes exact scaled dot-product softmax attention:
 *
 *   s_ij = c <q_i, k_j>,  LSE_i = ln sum_{valid j} exp(s_ij),
 *   P_ij = exp(s_ij - LSE_i) (exactly 0 for invalid j),  O_i = sum_j P_ij v_j,
 *
 * and, for the backward, dV = P^T dO, dS = P o (dO V^T - D) with
 * D_i = <dO_i, O_i>, dQ = c dS K, dK = c dS^T Q. The backward recomputes P
 * from the stored log-sum-exp instead of keeping it, the recomputation the
 * paper adopts for long sequences (Sec. V-B) in the manner of the attention
 * kernels it cites (Sec. II-C).
 *
 * Joint sequence of sample b (N = T + F*Hp*Wp tokens):
 *   positions [0, T)      text slot; the first clamp(text_len[b], 0, T) are
 *                         real caption tokens, the rest padding;
 *   positions [T, N)      video tokens, frame-major (frame, row, column).
 * Key j of sample b is valid iff
 *   (j >= T || j < clamp(text_len[b],0,T)) && (key_mask == NULL || key_mask[b*N+j] != 0).
 * Every token is a query, padded ones included. A query with no valid key gets
 * O = 0, LSE = -inf and dQ = 0. The token order inside the sequence does not
 * change any result (attention is equivariant in queries and invariant under
 * a joint permutation of keys and values), so the paper's interleaving of text
 * and visual embeddings is an ordering choice the caller may make freely.
 *
 * Conventions for every entry point
 *  - Tensors q, k, v, o, dout, dq, dk, dv: bf16, contiguous [B, N, H, D]
 *    (head_dim fastest), device memory, 16-byte aligned.
 *  - lse: fp32 [B, H, N], device memory, 16-byte aligned.
 *  - text_len: device int32 [B] or NULL (NULL means every text token is real).
 *  - key_mask: device uint8 [B, N] or NULL (NULL means no extra mask).
 *  - All memory is owned by the caller, workspaces included (except the fixed
 *    scratch array of vc_jointattn_fwd_noalloc). The library never
 *    allocates, frees or synchronises, keeps no per-call state, and only launches kernels on
 *    `stream` (a hipStream_t; NULL = the null stream). Outputs are
 *    overwritten, never accumulated into, and must not alias inputs.
 *  - Argument errors are reported synchronously, before anything is launched.
 *    Faults inside kernels surface at the caller's next synchronisation with
 *    the stream, as for any HIP kernel.
 *  - Thread-safe: the only shared state is a per-device property cache filled
 *    once (and the per-device scratch array of vc_jointattn_fwd_noalloc, whose
 *    concurrent calls on one device race).
 */
#ifndef VC_JOINTATTN_H
#define VC_JOINTATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Raised with every change of a signature, a struct, the meaning of an argument or a
 * documented result; the Python binding refuses a library that reports another
 * version. */
#define VC_JOINTATTN_ABI_VERSION 10

typedef enum vc_status {
  VC_OK = 0,
  VC_ERR_NULL = -1,        /* a required pointer is NULL                       */
  VC_ERR_SHAPE = -2,       /* a size is out of range or N overflows            */
  VC_ERR_HEAD_DIM = -3,    /* head_dim is not 64 or 128                        */
  VC_ERR_ALIGN = -4,       /* a tensor pointer is not 16-byte aligned          */
  VC_ERR_WORKSPACE = -5,   /* workspace NULL or smaller than required          */
  VC_ERR_DEVICE = -6,      /* no current HIP device, or it is not gfx950       */
  VC_ERR_HIP = -7,         /* a HIP launch reported an error                   */
  VC_ERR_UNSUPPORTED = -8, /* a requested mode is not available                */
  VC_ERR_ALIAS = -9,       /* an output is the same buffer as another output   */
  VC_ERR_SCRATCH = -10     /* the problem needs more scratch than the library's
                              fixed device array holds (no-allocation entry point) */
} vc_status;

/* Problem descriptor (passed by pointer, read only during the call). */
typedef struct vc_jointattn_desc {
  int32_t batch;          /* B >= 1                                             */
  int32_t heads;          /* H >= 1                                             */
  int32_t head_dim;       /* D, 64 or 128                                       */
  int32_t text_slot;      /* T >= 0: text tokens (padded) placed first          */
  int32_t frames;         /* F >= 1                                             */
  int32_t grid_h;         /* Hp >= 1: patch rows per frame                      */
  int32_t grid_w;         /* Wp >= 1: patch columns per frame                   */
  float softmax_scale;    /* c; <= 0 selects 1/sqrt(D)                          */
  int32_t deterministic;  /* 0: the joint backward computes dQ inside the
                             key-stationary kernel, adding it up with fp32
                             atomics (fastest; dQ may differ from run to run
                             by rounding). 1: a separate dQ pass, bitwise
                             reproducible. Other results never use atomics. */
} vc_jointattn_desc;

/* Version of this ABI (VC_JOINTATTN_ABI_VERSION). */
int vc_jointattn_abi_version(void);

/* Static text for a status code; never NULL. */
const char* vc_status_string(int status);

/* Joint sequence length N = T + F*Hp*Wp of a descriptor, or a negative
 * vc_status if the descriptor is invalid. Host only; touches no device. */
int64_t vc_jointattn_tokens(const vc_jointattn_desc* desc);

/* Bytes of device workspace the forward needs: a token-major copy of V
 * ([B,H,ceil(N/64)] tiles of D x 72 bf16), then room for the fp32 partial
 * results of up to 256 workgroups of 256 query rows (O, exponent base, sum),
 * used when the work's last round of workgroups on the device is split over
 * several workgroups to end early. 0 for an invalid descriptor. Host only. */
size_t vc_jointattn_fwd_workspace_bytes(const vc_jointattn_desc* desc);

/* Forward: o = softmax(c q k^T, masked) v and lse, as defined above.
 * Reads q, k, v, text_len, key_mask; writes o [B,N,H,D] bf16 and
 * lse [B,H,N] fp32 (natural log, scale included). `workspace` is caller-owned
 * device memory of at least vc_jointattn_fwd_workspace_bytes(desc) bytes,
 * 256-byte aligned; its contents on entry do not matter. Deterministic. */
vc_status vc_jointattn_fwd(const vc_jointattn_desc* desc,
                           const void* q, const void* k, const void* v,
                           const int32_t* text_len, const uint8_t* key_mask,
                           void* o, float* lse,
                           void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Forward without caller workspace, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): as vc_jointattn_fwd, with the workspace taken from a file-scope device
 * array of VC_JOINTATTN_NOALLOC_SCRATCH_BYTES inside the library, one per device,
 * held from the library's first use on that device until the process ends. The
 * call itself allocates and frees nothing; on its first call on a device it looks
 * up that device's copy of the array (with that device current) and keeps the
 * address. Problems whose vc_jointattn_fwd_workspace_bytes exceed the array return
 * VC_ERR_SCRATCH before anything is launched (256 MiB holds, at head_dim 128, up to
 * about 8.1e5 (sample, head, token) rows, e.g. 3 heads of 271k tokens; at head_dim 64
 * about 1.7e6). Every call on one device uses the same array: calls that overlap on a
 * device (other streams, other threads) race and must be serialised by the caller.
 * Nothing in the array needs clearing between calls: every byte read is written
 * first by the same call. Results are bitwise those of vc_jointattn_fwd.
 * ------------------------------------------------------------------------- */
#define VC_JOINTATTN_NOALLOC_SCRATCH_BYTES ((size_t)256 << 20)

vc_status vc_jointattn_fwd_noalloc(const vc_jointattn_desc* desc,
                                   const void* q, const void* k, const void* v,
                                   const int32_t* text_len, const uint8_t* key_mask,
                                   void* o, float* lse, void* stream);

/* Bytes of device workspace the backward needs: per query row fp32 -D and
 * LSE*log2(e) ([B,H,Npad], Npad = N rounded up to 64), token-major copies of
 * Q, dO and K (as for the forward's V; with desc->deterministic = 0 the same
 * region holds the fp32 dQ accumulator [B,N,H,D] instead), and room for fp32
 * partial dK, dV (or dQ) of up to 256 workgroups of 256 rows, used as in the
 * forward. 0 for an invalid descriptor. Host only. */
size_t vc_jointattn_bwd_workspace_bytes(const vc_jointattn_desc* desc);

/* Backward: dq, dk, dv (bf16 [B,N,H,D]) from q, k, v, the forward's o and lse,
 * and the upstream gradient dout. `workspace` is caller-owned device memory of
 * at least vc_jointattn_bwd_workspace_bytes(desc) bytes, 256-byte aligned; its
 * contents on entry do not matter. Masked keys get dk = dv = 0 exactly.
 * desc->deterministic = 1: equivalent to the three stage calls below in order;
 * no atomics, the result is bitwise reproducible run to run (on devices with a
 * different number of compute units the split of the last round of
 * workgroups, and so the summation order of its rows, differs).
 * desc->deterministic = 0: stage 1 (token-major copy of k only, none when the
 * fused pass carries every key), vc_jointattn_bwd_fused, then stage 3 over the
 * remaining keys; dk, dv are reproducible run to run, dq only up to the
 * rounding of its fp32 sums. When vc_jointattn_fused_dq_keys(desc) is 0 it
 * runs the deterministic stages instead. */
vc_status vc_jointattn_bwd(const vc_jointattn_desc* desc,
                           const void* q, const void* k, const void* v,
                           const void* o, const float* lse, const void* dout,
                           const int32_t* text_len, const uint8_t* key_mask,
                           void* dq, void* dk, void* dv,
                           void* workspace, size_t workspace_bytes, void* stream);

/* Backward stage 1: per query row, D_i = sum_d dO_id O_id and LSE_i*log2(e)
 * (fp32, padding rows made inert), the token-major copy of k and, when
 * desc->deterministic = 1, those of q and dout, all into the workspace.
 * Memory-bound. */
vc_status vc_jointattn_bwd_prepare(const vc_jointattn_desc* desc,
                                   const void* q, const void* k,
                                   const void* o, const float* lse, const void* dout,
                                   void* workspace, size_t workspace_bytes, void* stream);

/* Backward stage 2 (key-stationary): recompute P from the stage-1 LSE and write
 * dk = c dS^T Q and dv = P^T dO. Needs stage 1 on the same workspace, run with
 * desc->deterministic = 1; VC_ERR_UNSUPPORTED if desc->deterministic is 0. */
vc_status vc_jointattn_bwd_dkdv(const vc_jointattn_desc* desc,
                                const void* q, const void* k, const void* v,
                                const void* dout,
                                const int32_t* text_len, const uint8_t* key_mask,
                                void* dk, void* dv,
                                void* workspace, size_t workspace_bytes, void* stream);

/* Backward stage 3 (query-stationary): recompute P and dP and write
 * dq = c dS K. desc->deterministic = 1: over all keys; needs stage 1 on the
 * same workspace, independent of stage 2. desc->deterministic = 0: completes
 * the fused backward (stage 1, then vc_jointattn_bwd_fused, on the same
 * workspace): over the keys whose blocks did not add their share of dQ in the
 * fused pass, plus that pass's fp32 accumulator (when the fused pass carried
 * every key, the accumulator alone). */
vc_status vc_jointattn_bwd_dq(const vc_jointattn_desc* desc,
                              const void* q, const void* k, const void* v,
                              const void* dout,
                              const int32_t* text_len, const uint8_t* key_mask,
                              void* dq,
                              void* workspace, size_t workspace_bytes, void* stream);

/* Backward stage 2 of the fused backward (what vc_jointattn_bwd runs for
 * desc->deterministic = 0; this call does not read the flag): one
 * key-stationary pass recomputes P and dP and writes dk = c dS^T Q and
 * dv = P^T dO; the key blocks of a fixed leading fraction also add their share
 * of dq / c, dS K, to an fp32 accumulator in the workspace with atomics, so
 * that S and dP of those keys are computed once. Needs stage 1 on the same
 * workspace; stage 3 (vc_jointattn_bwd_dq with desc->deterministic = 0)
 * completes dq. */
/* Keys [0, K) whose share of dq the fused pass adds (vc_jointattn_bwd_fused);
 * stage 3 covers keys [K, N). K is the leading 65% of the 256-key blocks at
 * head_dim 128 and every key at head_dim 64 (the fastest splits measured),
 * never more than N; 0 when a sample's N*H*D elements reach 2^32 (the fused
 * pass addresses its accumulator with 32-bit offsets). Returns K, or a negative
 * vc_status if the descriptor is invalid. Host only. */
int64_t vc_jointattn_fused_dq_keys(const vc_jointattn_desc* desc);

vc_status vc_jointattn_bwd_fused(const vc_jointattn_desc* desc,
                                 const void* q, const void* k, const void* v,
                                 const void* dout,
                                 const int32_t* text_len, const uint8_t* key_mask,
                                 void* dk, void* dv,
                                 void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Spatial attention branch (Sec. III-B: the video sequence [B, F, L, ...]
 * regrouped as [B*F, L, ...], L = Hp*Wp, each frame on its own; the text tokens
 * join every frame's keys, Sec. V-B). Computed in
 * place on the joint layout: a video query of frame f attends to the valid text
 * keys and the valid keys of frame f, rows [T + f*L, T + (f+1)*L) (validity as
 * for the joint branch: text_len, key_mask). Text rows are not queries of this
 * branch: their o and dq are 0 and their lse -inf; text keys still receive dk,
 * dv from every frame. Same arguments and conventions as vc_jointattn_fwd /
 * vc_jointattn_bwd; the forward takes the joint forward workspace, the backward
 * its own (vc_spatialattn_bwd_workspace_bytes: the joint backward workspace plus
 * fp32 partial dk, dv of the text keys, whose work is split over several
 * workgroups). Each workgroup visits only the key tiles of the text and of its
 * own frames.
 * ------------------------------------------------------------------------- */

/* Bytes of backward workspace vc_spatialattn_bwd needs for this descriptor (at
 * least vc_jointattn_bwd_workspace_bytes), or 0 if the descriptor is invalid. */
size_t vc_spatialattn_bwd_workspace_bytes(const vc_jointattn_desc* desc);

/* Spatial forward: o [B,N,H,D] bf16 and lse [B,H,N] fp32 (natural log). */
vc_status vc_spatialattn_fwd(const vc_jointattn_desc* desc,
                             const void* q, const void* k, const void* v,
                             const int32_t* text_len, const uint8_t* key_mask,
                             void* o, float* lse,
                             void* workspace, size_t workspace_bytes, void* stream);

/* Spatial backward: dq, dk, dv from q, k, v, the spatial forward's o and lse, and
 * dout; workspace of vc_spatialattn_bwd_workspace_bytes (smaller: VC_ERR_WORKSPACE,
 * nothing launched). desc->deterministic = 1: separate dK/dV and dQ passes, bitwise
 * reproducible, no atomics. desc->deterministic = 0: one key-stationary pass also
 * adds every key block's share of dq to an fp32 accumulator with atomics (a video
 * query row gets the shares of its frame's key blocks and of the text block); dk,
 * dv are reproducible run to run, dq only up to the rounding of its fp32 sums.
 * When a sample's N*H*D elements reach 2^32 the separate passes run for either
 * value of the flag. */
vc_status vc_spatialattn_bwd(const vc_jointattn_desc* desc,
                             const void* q, const void* k, const void* v,
                             const void* o, const float* lse, const void* dout,
                             const int32_t* text_len, const uint8_t* key_mask,
                             void* dq, void* dk, void* dv,
                             void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Temporal attention branch (Sec. III-B: besides the full-sequence branch the
 * block attends over the video sequence [B, F, L, ...] regrouped as
 * [B*L, F, ...], L = Hp*Wp tokens per frame; the branch outputs are added).
 * It is computed in place on the joint layout: the video token of frame f at
 * spatial position l, row T + f*L + l, attends to the F rows T + f'*L + l,
 * f' = 0..F-1, with key_mask (NULL = none) applied to those keys; a query with
 * no valid key gets O = 0, LSE = -inf. Text rows take no part: their o, dq, dk,
 * dv are written as 0 and their lse as -inf. text_len is not used. Requires
 * F <= 144 (VC_ERR_SHAPE otherwise; the paper's longest clip has 144 frames,
 * Sec. VI-D): up to 32 frames one matrix-core block packs several positions,
 * beyond that a workgroup takes one position at a time, frames in blocks of 32.
 * Tensor conventions as above; results are deterministic and no atomics are used.
 * ------------------------------------------------------------------------- */

/* Temporal forward: writes o [B,N,H,D] bf16 and lse [B,H,N] fp32 (natural log).
 * Needs no workspace. */
vc_status vc_temporalattn_fwd(const vc_jointattn_desc* desc,
                              const void* q, const void* k, const void* v,
                              const uint8_t* key_mask,
                              void* o, float* lse, void* stream);

/* Temporal forward with the branch sum fused into its epilogue: as
 * vc_temporalattn_fwd, and in the same pass out = o_joint + o_spatial + o over
 * every row (this branch's o is 0 on text rows), with the arithmetic of
 * vc_branchsum, so `out` is bitwise what vc_branchsum(o_joint, o_spatial, o)
 * would write. o_joint or o_spatial may be NULL (zero); out may be o_joint or
 * o_spatial (in-place accumulation) but not o (VC_ERR_ALIAS). */
vc_status vc_temporalattn_fwd_sum(const vc_jointattn_desc* desc,
                                  const void* q, const void* k, const void* v,
                                  const uint8_t* key_mask,
                                  const void* o_joint, const void* o_spatial,
                                  void* o, float* lse, void* out, void* stream);

/* Bytes of device workspace the temporal backward was documented to need (per
 * row fp32 -D and LSE*log2(e), [B,H,Npad]); 0 for an invalid descriptor. Host
 * only. Kept for callers that size the argument with it: the backward forms both
 * values inside its kernels and neither reads nor checks the workspace (it may be
 * NULL). */
size_t vc_temporalattn_bwd_workspace_bytes(const vc_jointattn_desc* desc);

/* Temporal backward: dq, dk, dv from q, k, v, the temporal forward's o and lse
 * and dout. `workspace` and `workspace_bytes` are not used (any value, NULL
 * included). */
vc_status vc_temporalattn_bwd(const vc_jointattn_desc* desc,
                              const void* q, const void* k, const void* v,
                              const void* o, const float* lse, const void* dout,
                              const uint8_t* key_mask,
                              void* dq, void* dk, void* dv,
                              void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Branch sum (Sec. III-B: a block's attention output is the element-wise sum
 * of its three branch results, spatial, temporal and joint). The backward of the sum needs no kernel: every branch's backward
 * takes the same dout.
 * ------------------------------------------------------------------------- */

/* out = o_joint + o_spatial + o_temporal, element-wise over [B,N,H,D] bf16: each
 * element is summed in fp32 in that order and rounded once to bf16 (nearest
 * even). Any input may be NULL (a branch the model does not run counts as
 * zero), but not all three (VC_ERR_NULL); out may be one of the inputs. */
vc_status vc_branchsum(const vc_jointattn_desc* desc,
                       const void* o_joint, const void* o_spatial, const void* o_temporal,
                       void* out, void* stream);

/* ---------------------------------------------------------------------------
 * Activation offload (Sec. V-B: saved activations swapped to host memory on a
 * separate stream, overlapped with computation, as a substitute for
 * recomputation in selected layers; compared in Sec. VI-D). An engine owns one
 * copy stream (default priority) and two events; copies run on it and never
 * block the host.
 *  - Ordering: a store or load starts only after all work the caller queued on
 *    `stream` before the call (so a tensor a kernel writes on `stream` can be
 *    stored right after the launch). vc_offload_wait makes `stream` wait for
 *    every copy issued so far: a stored device buffer may be overwritten, and a
 *    loaded one read, on `stream` only after that wait.
 *  - Memory: host buffers must be pinned (hipHostMalloc, or torch's
 *    pin_memory); device buffers must be device memory of the engine's device.
 *    Each [ptr, ptr + bytes) must lie inside one allocation. Otherwise
 *    VC_ERR_UNSUPPORTED and nothing is issued. A call from another current
 *    device than the engine's: VC_ERR_DEVICE.
 *  - An engine is not thread-safe; use one per thread. bytes = 0 is a no-op.
 * ------------------------------------------------------------------------- */
typedef struct vc_offload vc_offload;

/* Creates an engine on the current device; *out receives it (NULL on error). */
vc_status vc_offload_create(vc_offload** out);

/* Waits for the engine's copies to finish, then frees it. */
vc_status vc_offload_destroy(vc_offload* h);

/* Device -> pinned host copy of `bytes` bytes, ordered after `stream`'s work. */
vc_status vc_offload_store(vc_offload* h, void* host_dst, const void* dev_src, size_t bytes,
                           void* stream);

/* Pinned host -> device copy of `bytes` bytes, ordered after `stream`'s work. */
vc_status vc_offload_load(vc_offload* h, void* dev_dst, const void* host_src, size_t bytes,
                          void* stream);

/* Makes `stream` wait (on the device) for every copy issued so far. */
vc_status vc_offload_wait(vc_offload* h, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* VC_JOINTATTN_H */
