// Forward joint text-video attention for gfx950.
//
// One workgroup of four waves owns 128 queries of one (sample, head); each
// wave owns 32 of them. Keys and values stream through LDS in tiles of 64.
// The wave computes the transposed score block S^T = K Q^T with the matrix
// cores (32x32x16 bf16), so each lane's accumulator column is one query:
// the running maximum and sum of the online softmax are per-lane scalars and
// need one exchange between the two wave halves per tile. P^T leaves the
// accumulator already laid out as the B operand of O^T += V^T P^T, so
// probabilities never go through LDS. V is stored transposed in LDS for that
// product. The log-sum-exp is kept for the recomputing backward.
#include "common.hpp"

namespace vcja {
namespace {

constexpr int kBM = 128;  // queries per workgroup
constexpr int kBN = 64;   // keys per tile

template <int D>
__global__ __launch_bounds__(256, 1) void fwd_kernel(FwdArgs a) {
  constexpr int KS = D + 8;    // K row stride in LDS (bf16), padded against bank conflicts
  constexpr int VS = kBN + 4;  // V^T row stride in LDS (bf16)
  __shared__ __attribute__((aligned(16))) __bf16 ks_lds[kBN * KS];
  __shared__ __attribute__((aligned(16))) __bf16 vt_lds[D * VS];

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
  const int qi = blockIdx.x * kBM + w * 32 + l32;

  // Q^T as the B operand: lane holds query qi, dims 16*ks + 8*hi .. +7.
  bf16x8 qf[D / 16];
  if (qi < N) {
    const __bf16* qp = a.q + base + (size_t)qi * tok + 8 * hi;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) qf[ks] = *(const bf16x8*)(qp + 16 * ks);
  } else {
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) qf[ks] = zero_bf16x8();
  }

  f32x16 oacc[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) oacc[i] = zero_f32x16();
  float m = -INFINITY;  // running max of scaled scores, log2 units
  float l = 0.0f;       // running sum of this lane's half

  int tl = a.T;
  if (a.text_len) tl = min(max(a.text_len[b], 0), a.T);
  const uint8_t* km = a.key_mask ? a.key_mask + (size_t)b * N : nullptr;
  const int ntiles = (N + kBN - 1) / kBN;

  for (int kt = 0; kt < ntiles; ++kt) {
    const int k0 = kt * kBN;
    // A tile made only of padded text keys contributes nothing.
    if (!km && k0 >= tl && k0 + kBN <= a.T) continue;
    __syncthreads();
    // K tile, row-major.
    for (int c = tid; c < kBN * D / 8; c += 256) {
      const int kr = c / (D / 8);
      const int col = (c % (D / 8)) * 8;
      const int key = k0 + kr;
      bf16x8 val = zero_bf16x8();
      if (key < N) val = *(const bf16x8*)(a.k + base + (size_t)key * tok + col);
      *(bf16x8*)&ks_lds[kr * KS + col] = val;
    }
    // V tile, transposed: thread takes 4 keys x 8 dims.
    for (int g = tid; g < (kBN / 4) * (D / 8); g += 256) {
      const int kg = g / (D / 8);
      const int dg = g % (D / 8);
      bf16x8 r[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = k0 + 4 * kg + i;
        r[i] = zero_bf16x8();
        if (key < N) r[i] = *(const bf16x8*)(a.v + base + (size_t)key * tok + 8 * dg);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        bf16x4 t = {r[0][e], r[1][e], r[2][e], r[3][e]};
        *(bf16x4*)&vt_lds[(8 * dg + e) * VS + 4 * kg] = t;
      }
    }
    __syncthreads();

    // S^T = K Q^T for two 32-key blocks.
    f32x16 s[kBN / 32];
#pragma unroll
    for (int kb = 0; kb < kBN / 32; ++kb) {
      s[kb] = zero_f32x16();
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) {
        bf16x8 af = *(const bf16x8*)&ks_lds[(kb * 32 + l32) * KS + 16 * ks + 8 * hi];
        s[kb] = mfma32(af, qf[ks], s[kb]);
      }
    }

    const bool need_mask = km || (tl < a.T && k0 < a.T && k0 + kBN > tl) || (k0 + kBN > N);
    if (need_mask) {
#pragma unroll
      for (int kb = 0; kb < kBN / 32; ++kb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = k0 + kb * 32 + acc_row(r, hi);
          bool ok = key < N && (key >= a.T || key < tl);
          if (ok && km) ok = km[key] != 0;
          if (!ok) s[kb][r] = -INFINITY;
        }
      }
    }

    // Online softmax; this lane's column is query qi.
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < kBN / 32; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
    mx = fmaxf(mx, swap_halves(mx));
    const float m_new = fmaxf(m, mx * a.scale_log2);
    const float m_use = (m_new == -INFINITY) ? 0.0f : m_new;
    const float alpha = fast_exp2(m - m_use);
    m = m_new;
    l *= alpha;
#pragma unroll
    for (int i = 0; i < D / 32; ++i) oacc[i] *= alpha;

    float p[kBN / 32][16];
#pragma unroll
    for (int kb = 0; kb < kBN / 32; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        p[kb][r] = fast_exp2(fmaf(s[kb][r], a.scale_log2, -m_use));
        l += p[kb][r];
      }

    // O^T += V^T P^T. Register r of the S^T block maps to key 8*(r/4) + 4*hi + r%4, so the
    // operand pair (lane half hi, element t) of k-step st stands for key
    // 16*st + 8*(t/4) + 4*hi + t%4; V^T is read in that order.
#pragma unroll
    for (int kb = 0; kb < kBN / 32; ++kb) {
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        const bf16x8 pb = to_bf16x8(&p[kb][8 * st]);
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          const __bf16* vp = &vt_lds[(db * 32 + l32) * VS + kb * 32 + 16 * st + 4 * hi];
          const bf16x8 af = cat4(*(const bf16x4*)vp, *(const bf16x4*)(vp + 8));
          oacc[db] = mfma32(af, pb, oacc[db]);
        }
      }
    }
  }

  const float lt = l + swap_halves(l);
  const float inv = lt > 0.0f ? 1.0f / lt : 0.0f;
  if (qi < N) {
    __bf16* op = a.o + base + (size_t)qi * tok;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        bf16x4 t = {(__bf16)(oacc[db][4 * j + 0] * inv), (__bf16)(oacc[db][4 * j + 1] * inv),
                    (__bf16)(oacc[db][4 * j + 2] * inv), (__bf16)(oacc[db][4 * j + 3] * inv)};
        *(bf16x4*)(op + db * 32 + 8 * j + 4 * hi) = t;
      }
    if (hi == 0)
      a.lse[((size_t)b * a.H + h) * N + qi] = lt > 0.0f ? (m + __log2f(lt)) * kLn2 : -INFINITY;
  }
}

}  // namespace

hipError_t launch_fwd(const FwdArgs& a, int head_dim, hipStream_t s) {
  dim3 grid((a.N + kBM - 1) / kBM, a.H, a.B);
  if (head_dim == 128)
    hipLaunchKernelGGL(fwd_kernel<128>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(fwd_kernel<64>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace vcja
