// Backward joint text-video attention for gfx950.
//
// Stage 1 (prepare): D_i = <dO_i, O_i> in fp32, and a zeroed fp32 dQ accumulator.
// Stage 2 (main): one workgroup of four waves owns 128 keys of one (sample,
//   head), each wave 32 of them, with K and V of its keys held in registers and
//   dK^T, dV^T accumulated in registers. It walks over all query tiles of 64:
//   recomputes S = Q K^T and P = exp(S c - LSE) with the matrix cores, forms
//   dP = dO V^T and dS = P o (dP - D), and accumulates dV^T += dO^T P and
//   dK^T += Q^T dS straight from the accumulator layout (lane column = key).
//   dS goes through LDS once so the workgroup can form the dQ contribution of
//   its 128 keys, dQ += c dS K, which is added to the fp32 accumulator with
//   atomics.
// Stage 3 (finish): dQ accumulator -> bf16.
#include "common.hpp"

namespace vcja {
namespace {

constexpr int kBKV = 128;  // keys per workgroup
constexpr int kBQ = 64;    // queries per inner tile

template <int D>
__global__ __launch_bounds__(256) void bwd_prepare_kernel(const __bf16* __restrict__ o,
                                                          const __bf16* __restrict__ dout,
                                                          float* __restrict__ dd, float* __restrict__ dq_acc,
                                                          int B, int H, int N) {
  constexpr int CPR = D / 8;  // 16-byte chunks per (token, head) row
  const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t rows = (size_t)B * N * H;
  const size_t row = gid / CPR;
  const int chunk = (int)(gid % CPR);
  float sum = 0.0f;
  if (row < rows) {
    const bf16x8 x = *(const bf16x8*)(o + row * D + chunk * 8);
    const bf16x8 y = *(const bf16x8*)(dout + row * D + chunk * 8);
#pragma unroll
    for (int e = 0; e < 8; ++e) sum = fmaf((float)x[e], (float)y[e], sum);
    f32x4 z = {0.f, 0.f, 0.f, 0.f};
    *(f32x4*)(dq_acc + row * D + chunk * 8) = z;
    *(f32x4*)(dq_acc + row * D + chunk * 8 + 4) = z;
  }
#pragma unroll
  for (int off = 1; off < CPR; off <<= 1) sum += __shfl_xor(sum, off, 64);
  if (row < rows && chunk == 0) {
    const int h = (int)(row % H);
    const size_t bn = row / H;
    const int n = (int)(bn % N);
    const int b = (int)(bn / N);
    dd[((size_t)b * H + h) * N + n] = sum;
  }
}

__global__ __launch_bounds__(256) void bwd_finish_kernel(const float* __restrict__ acc, __bf16* __restrict__ dq,
                                                         size_t n8) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n8) return;
  const f32x4 x0 = *(const f32x4*)(acc + 8 * i);
  const f32x4 x1 = *(const f32x4*)(acc + 8 * i + 4);
  bf16x8 r = {(__bf16)x0[0], (__bf16)x0[1], (__bf16)x0[2], (__bf16)x0[3],
              (__bf16)x1[0], (__bf16)x1[1], (__bf16)x1[2], (__bf16)x1[3]};
  *(bf16x8*)(dq + 8 * i) = r;
}

// Loads rows [q0, q0+64) of a [B,N,H,D] tensor slice into LDS twice: row-major
// (stride D+8) and transposed (stride kBQ+4). Each thread takes 4 rows x 8 dims.
template <int D>
__device__ __forceinline__ void load_tile_both(const __bf16* __restrict__ src, size_t base, size_t tok, int q0,
                                               int N, __bf16* rowmaj, __bf16* trans, int tid) {
  constexpr int RS = D + 8;
  constexpr int TS = kBQ + 4;
  for (int g = tid; g < (kBQ / 4) * (D / 8); g += 256) {
    const int rg = g / (D / 8);
    const int dg = g % (D / 8);
    bf16x8 r[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = q0 + 4 * rg + i;
      r[i] = zero_bf16x8();
      if (row < N) r[i] = *(const bf16x8*)(src + base + (size_t)row * tok + 8 * dg);
      *(bf16x8*)&rowmaj[(4 * rg + i) * RS + 8 * dg] = r[i];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      bf16x4 t = {r[0][e], r[1][e], r[2][e], r[3][e]};
      *(bf16x4*)&trans[(8 * dg + e) * TS + 4 * rg] = t;
    }
  }
}

template <int D>
__global__ __launch_bounds__(256, 1) void bwd_main_kernel(BwdArgs a) {
  constexpr int RS = D + 8;      // row-major Q / dO stride
  constexpr int TS = kBQ + 4;    // transposed Q / dO stride
  constexpr int SS = kBKV + 8;   // dS stride
  __shared__ __attribute__((aligned(16))) __bf16 q_lds[kBQ * RS];
  __shared__ __attribute__((aligned(16))) __bf16 do_lds[kBQ * RS];
  __shared__ __attribute__((aligned(16))) __bf16 qt_lds[D * TS];
  __shared__ __attribute__((aligned(16))) __bf16 dot_lds[D * TS];
  __shared__ __attribute__((aligned(16))) __bf16 ds_lds[kBQ * SS];
  __shared__ float lse_lds[kBQ];
  __shared__ float dd_lds[kBQ];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int l32 = lane & 31;
  const int hi = lane >> 5;
  const int h = blockIdx.y;
  const int b = blockIdx.z;
  const int N = a.N;
  const size_t tok = (size_t)a.H * D;
  const size_t base = (size_t)b * N * tok + (size_t)h * D;
  const size_t bh = (size_t)b * a.H + h;
  const int kbase = blockIdx.x * kBKV;
  const int key = kbase + w * 32 + l32;  // this lane's key (accumulator column)

  int tl = a.T;
  if (a.text_len) tl = min(max(a.text_len[b], 0), a.T);
  bool valid = key < N && (key >= a.T || key < tl);
  if (valid && a.key_mask) valid = a.key_mask[(size_t)b * N + key] != 0;

  if (!__syncthreads_or(valid)) {
    // No valid key in this workgroup: its dK, dV are zero and it adds nothing to dQ.
    if (key < N) {
      bf16x8 z = zero_bf16x8();
      for (int c = 0; c < D / 8; ++c) {
        *(bf16x8*)(a.dk + base + (size_t)key * tok + 8 * c) = z;
        *(bf16x8*)(a.dv + base + (size_t)key * tok + 8 * c) = z;
      }
    }
    return;
  }

  // K, V of this lane's key as B operands (dims 16*ks + 8*hi .. +7).
  bf16x8 kf[D / 16], vf[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    kf[ks] = zero_bf16x8();
    vf[ks] = zero_bf16x8();
    if (key < N) {
      kf[ks] = *(const bf16x8*)(a.k + base + (size_t)key * tok + 16 * ks + 8 * hi);
      vf[ks] = *(const bf16x8*)(a.v + base + (size_t)key * tok + 16 * ks + 8 * hi);
    }
  }

  // dQ blocks owned by this wave: (query block qb, dim slice dsl) of 32x32.
  constexpr int kDqBlocks = (kBQ / 32) * (D / 32) / 4;  // per wave: 2 for D=128, 1 for D=64
  const int dsl = (D == 128) ? w : (w & 1);
  const int qb_first = (D == 128) ? 0 : (w >> 1);
  // K as the B operand of dQ = dS K: lane holds dim dsl*32 + l32, keys 16*ks + 8*hi .. +7.
  bf16x8 ktf[kBKV / 16];
#pragma unroll
  for (int ks = 0; ks < kBKV / 16; ++ks) {
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const int kk = kbase + 16 * ks + 8 * hi + t;
      ktf[ks][t] = (kk < N) ? a.k[base + (size_t)kk * tok + dsl * 32 + l32] : (__bf16)0.0f;
    }
  }

  f32x16 dk_acc[D / 32], dv_acc[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) {
    dk_acc[i] = zero_f32x16();
    dv_acc[i] = zero_f32x16();
  }

  const int nqt = (N + kBQ - 1) / kBQ;
  for (int qt = 0; qt < nqt; ++qt) {
    const int q0 = qt * kBQ;
    __syncthreads();
    load_tile_both<D>(a.q, base, tok, q0, N, q_lds, qt_lds, tid);
    load_tile_both<D>(a.dout, base, tok, q0, N, do_lds, dot_lds, tid);
    if (tid < kBQ) {
      const int row = q0 + tid;
      float l2 = INFINITY, dv = 0.0f;
      if (row < N) {
        const float x = a.lse[bh * N + row];
        l2 = (x == -INFINITY) ? INFINITY : x * kLog2e;  // rows without keys: P = 0
        dv = a.dd[bh * N + row];
      }
      lse_lds[tid] = l2;
      dd_lds[tid] = dv;
    }
    __syncthreads();

#pragma unroll
    for (int qb = 0; qb < kBQ / 32; ++qb) {
      f32x16 s = zero_f32x16(), dp = zero_f32x16();
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) {
        const bf16x8 qa = *(const bf16x8*)&q_lds[(qb * 32 + l32) * RS + 16 * ks + 8 * hi];
        s = mfma32(qa, kf[ks], s);
      }
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) {
        const bf16x8 da = *(const bf16x8*)&do_lds[(qb * 32 + l32) * RS + 16 * ks + 8 * hi];
        dp = mfma32(da, vf[ks], dp);
      }
      float p[16], ds[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ql = qb * 32 + acc_row(r, hi);
        p[r] = valid ? fast_exp2(fmaf(s[r], a.scale_log2, -lse_lds[ql])) : 0.0f;
        ds[r] = p[r] * (dp[r] - dd_lds[ql]);
      }
      // Register r holds query row 8*(r/4) + 4*hi + r%4; operand element t of k-step st
      // stands for query 16*st + 8*(t/4) + 4*hi + t%4, and Q^T / dO^T are read in that order.
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        const bf16x8 pb = to_bf16x8(&p[8 * st]);
        const bf16x8 sb = to_bf16x8(&ds[8 * st]);
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          const int off = (db * 32 + l32) * TS + qb * 32 + 16 * st + 4 * hi;
          const bf16x8 doa = cat4(*(const bf16x4*)&dot_lds[off], *(const bf16x4*)&dot_lds[off + 8]);
          dv_acc[db] = mfma32(doa, pb, dv_acc[db]);
          const bf16x8 qa = cat4(*(const bf16x4*)&qt_lds[off], *(const bf16x4*)&qt_lds[off + 8]);
          dk_acc[db] = mfma32(qa, sb, dk_acc[db]);
        }
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ql = qb * 32 + acc_row(r, hi);
        ds_lds[ql * SS + w * 32 + l32] = (__bf16)ds[r];
      }
    }
    __syncthreads();

    // dQ contribution of this workgroup's keys for the tile.
#pragma unroll
    for (int i = 0; i < kDqBlocks; ++i) {
      const int qb = qb_first + i;
      f32x16 acc = zero_f32x16();
#pragma unroll
      for (int ks = 0; ks < kBKV / 16; ++ks) {
        const bf16x8 sa = *(const bf16x8*)&ds_lds[(qb * 32 + l32) * SS + 16 * ks + 8 * hi];
        acc = mfma32(sa, ktf[ks], acc);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int qrow = q0 + qb * 32 + acc_row(r, hi);
        if (qrow < N) unsafeAtomicAdd(a.dq_acc + ((size_t)b * N + qrow) * tok + (size_t)h * D + dsl * 32 + l32,
                                      acc[r] * a.scale);
      }
    }
  }

  if (key < N) {
    __bf16* dkp = a.dk + base + (size_t)key * tok;
    __bf16* dvp = a.dv + base + (size_t)key * tok;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        bf16x4 tk = {(__bf16)(dk_acc[db][4 * j + 0] * a.scale), (__bf16)(dk_acc[db][4 * j + 1] * a.scale),
                     (__bf16)(dk_acc[db][4 * j + 2] * a.scale), (__bf16)(dk_acc[db][4 * j + 3] * a.scale)};
        bf16x4 tv = {(__bf16)dv_acc[db][4 * j + 0], (__bf16)dv_acc[db][4 * j + 1], (__bf16)dv_acc[db][4 * j + 2],
                     (__bf16)dv_acc[db][4 * j + 3]};
        *(bf16x4*)(dkp + db * 32 + 8 * j + 4 * hi) = tk;
        *(bf16x4*)(dvp + db * 32 + 8 * j + 4 * hi) = tv;
      }
  }
}

}  // namespace

hipError_t launch_bwd_prepare(const __bf16* o, const __bf16* dout, float* dd, float* dq_acc, int B, int H, int N,
                              int head_dim, hipStream_t s) {
  const size_t threads = (size_t)B * N * H * (head_dim / 8);
  dim3 grid((unsigned)((threads + 255) / 256));
  if (head_dim == 128)
    hipLaunchKernelGGL(bwd_prepare_kernel<128>, grid, dim3(256), 0, s, o, dout, dd, dq_acc, B, H, N);
  else
    hipLaunchKernelGGL(bwd_prepare_kernel<64>, grid, dim3(256), 0, s, o, dout, dd, dq_acc, B, H, N);
  return hipGetLastError();
}

hipError_t launch_bwd_main(const BwdArgs& a, int head_dim, hipStream_t s) {
  dim3 grid((a.N + kBKV - 1) / kBKV, a.H, a.B);
  if (head_dim == 128)
    hipLaunchKernelGGL(bwd_main_kernel<128>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(bwd_main_kernel<64>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_bwd_finish(const float* dq_acc, __bf16* dq, int B, int H, int N, int head_dim, hipStream_t s) {
  const size_t n8 = (size_t)B * N * H * head_dim / 8;
  dim3 grid((unsigned)((n8 + 255) / 256));
  hipLaunchKernelGGL(bwd_finish_kernel, grid, dim3(256), 0, s, dq_acc, dq, n8);
  return hipGetLastError();
}

}  // namespace vcja
