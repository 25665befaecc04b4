// Device-side types and helpers shared by the joint-attention kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace vcja {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// One 32x32x16 bf16 matrix-core step: acc += A(32x16) * B(16x32).
// Lane l supplies A[l%32][8*(l/32) + t] and B[8*(l/32) + t][l%32], t = 0..7;
// it receives acc[r] = C[8*(r/4) + 4*(l/32) + r%4][l%32], r = 0..15.
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Row of the 32x32 accumulator held in register r by a lane of half `hi`.
__device__ __forceinline__ int acc_row(int r, int hi) { return 8 * (r >> 2) + 4 * hi + (r & 3); }

// Hardware 2^x (v_exp_f32); -inf -> 0.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ bf16x8 cat4(bf16x4 a, bf16x4 b) {
  return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// Eight fp32 -> bf16 (round to nearest even), packed as an MFMA operand.
__device__ __forceinline__ bf16x8 to_bf16x8(const float* x) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = (__bf16)x[i];
  return r;
}

__device__ __forceinline__ bf16x8 zero_bf16x8() {
  bf16x8 z;
#pragma unroll
  for (int i = 0; i < 8; ++i) z[i] = (__bf16)0.0f;
  return z;
}

__device__ __forceinline__ f32x16 zero_f32x16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.0f;
  return z;
}

// Value of lane l^32 (the other half of the wave).
__device__ __forceinline__ float swap_halves(float x) { return __shfl_xor(x, 32, 64); }

// Kernel arguments. Token stride is H*D elements ([B, N, H, D] layout).
struct FwdArgs {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  const int32_t* text_len;
  const uint8_t* key_mask;
  __bf16* o;
  float* lse;
  int B, H, N, T;
  float scale_log2;  // softmax scale times log2(e)
};

struct BwdArgs {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  const __bf16* dout;
  const float* lse;
  const float* dd;      // D = rowsum(dO o O), [B, H, N]
  const int32_t* text_len;
  const uint8_t* key_mask;
  __bf16* dk;
  __bf16* dv;
  float* dq_acc;        // [B, N, H, D] fp32
  int B, H, N, T;
  float scale;          // softmax scale
  float scale_log2;     // scale * log2(e)
};

}  // namespace vcja

// Host-side launchers (defined in the .hip kernel files).
namespace vcja {
hipError_t launch_fwd(const FwdArgs& a, int head_dim, hipStream_t s);
hipError_t launch_bwd_prepare(const __bf16* o, const __bf16* dout, float* dd, float* dq_acc, int B, int H,
                              int N, int head_dim, hipStream_t s);
hipError_t launch_bwd_main(const BwdArgs& a, int head_dim, hipStream_t s);
hipError_t launch_bwd_finish(const float* dq_acc, __bf16* dq, int B, int H, int N, int head_dim,
                             hipStream_t s);
}  // namespace vcja
