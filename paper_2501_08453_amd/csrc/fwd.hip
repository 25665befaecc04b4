// Forward joint text-video attention for gfx950.
//
// One workgroup of eight waves owns 256 queries of one (sample, head); each
// wave owns 32 of them, held in registers. Keys stream through LDS as
// row-major tiles of 64 (rows padded by 16 bytes) and values as
// transposed token tiles (prepared by a reformatting pass), both copied
// asynchronously global -> LDS into a two-stage ring so the next tile lands
// while the current one is computed; one barrier per tile. All eight waves
// share each tile.
//
// The wave computes the transposed score block S^T = K Q^T with 32x32x16 bf16
// matrix-core steps, so each lane's accumulator column is one query: the
// running maximum and sum of the online softmax are per-lane scalars that need
// one exchange between the two wave halves per tile. P^T leaves the
// accumulator already laid out as the B operand of O^T += V^T P^T, so
// probabilities never go through LDS. The exponent base is only raised when a
// tile's maximum exceeds it by more than 2^8, so the O^T rescale is rare
// (probabilities stay below 256, exact in the bf16 exponent range). The
// log-sum-exp is kept for the recomputing backward.
#include "common.hpp"

namespace vcja {
namespace {

constexpr int kWaves = 8;
constexpr int kBM = 32 * kWaves;  // queries per workgroup
constexpr int kBN = kTileTok;     // keys per tile
constexpr float kRescaleSlack = 8.0f;  // log2 units

template <int D>
__global__ __launch_bounds__(64 * kWaves, 1) void fwd_kernel(FwdArgs a) {
  constexpr int KT = RowTile<D>::kBytes;        // K tile bytes
  constexpr int KS = RowTile<D>::kStride;       // K row stride
  constexpr int VTB = (int)tile_elems(D) * 2;   // V^T tile bytes
  constexpr int STAGE = KT + VTB;
  constexpr int KCOPIES = RowTile<D>::kCopies;  // 1 KiB wave copies per tile
  constexpr int VCOPIES = VTB / 1024;
  static_assert(VTB % 1024 == 0, "transposed tile must be whole wave copies");
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index (uniform)
  const int l32 = lane & 31;
  const int hi = lane >> 5;
  const int h = blockIdx.y;
  const int b = blockIdx.z;
  const int N = a.N;
  const size_t tok = (size_t)a.H * D;
  const size_t base = (size_t)b * N * tok + (size_t)h * D;
  const __bf16* vt_bh = a.vt + ((size_t)b * a.H + h) * a.ntile * tile_elems(D);
  const int qi = blockIdx.x * kBM + w * 32 + l32;

  // Q^T as the B operand: lane holds query qi, dims 16*ks + 8*hi .. +7.
  bf16x8 qf[D / 16];
  {
    const __bf16* qp = a.q + base + (size_t)min(qi, N - 1) * tok + 8 * hi;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) qf[ks] = *(const bf16x8*)(qp + 16 * ks);
  }

  f32x16 oacc[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) oacc[i] = zero_f32x16();
  float m = -INFINITY;  // exponent base (scaled scores, log2 units)
  float l = 0.0f;       // running sum of this lane's half

  int tl = a.T;
  if (a.text_len) tl = min(max(a.text_len[b], 0), a.T);
  const uint8_t* km = a.key_mask ? a.key_mask + (size_t)b * N : nullptr;
  // A tile made only of padded text keys contributes nothing and is skipped.
  auto next_tile = [&](int kt) {
    if (!km)
      while (kt < a.ntile && kt * kBN >= tl && kt * kBN + kBN <= a.T) ++kt;
    return kt;
  };
  // Copies tile kt (K rows, V^T tile) into stage st. K rows past N repeat row N-1 and
  // are masked.
  auto issue = [&](int kt, int st) {
    VC_LDS char* sk = (VC_LDS char*)smem + st * STAGE;
    for (int idx = w; idx < KCOPIES; idx += kWaves) copy_row_tile<D>(a.k + base, tok, kt * kBN, N, sk, idx, lane);
    const __bf16* vsrc = vt_bh + (size_t)kt * tile_elems(D);
    for (int idx = w; idx < VCOPIES; idx += kWaves) copy16_to_lds(vsrc + idx * 512 + lane * 8, sk + KT + idx * 1024);
  };

  int kt = next_tile(0);
  if (kt < a.ntile) issue(kt, 0);
  int st = 0;
  while (kt < a.ntile) {
    const int kn = next_tile(kt + 1);
    wait_all_memory();
    __syncthreads();  // stage st holds tile kt; every wave is done with stage st^1
    if (kn < a.ntile) issue(kn, st ^ 1);
    const VC_LDS char* ks_lds = (const VC_LDS char*)smem + st * STAGE;
    const VC_LDS char* vt_lds = ks_lds + KT;
    const int k0 = kt * kBN;

    // S^T = K Q^T for two 32-key blocks.
    f32x16 s[kBN / 32];
#pragma unroll
    for (int kb = 0; kb < kBN / 32; ++kb) {
      s[kb] = zero_f32x16();
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) {
        const bf16x8 af = *(const VC_LDS bf16x8*)(ks_lds + (kb * 32 + l32) * KS + (2 * ks + hi) * 16);
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
    mx = fmaxf(mx, swap_halves(mx)) * a.scale_log2;
    const bool raise = mx > m + kRescaleSlack;
    if (__any(raise)) {
      const float m_new = raise ? mx : m;
      const float alpha = raise ? fast_exp2(m - m_new) : 1.0f;  // 0 when m was -inf
      m = m_new;
      l *= alpha;
#pragma unroll
      for (int i = 0; i < D / 32; ++i) oacc[i] *= alpha;
    }
    const float m_use = (m == -INFINITY) ? 0.0f : m;

    float p[kBN / 32][16];
#pragma unroll
    for (int kb = 0; kb < kBN / 32; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        p[kb][r] = fast_exp2(fmaf(s[kb][r], a.scale_log2, -m_use));
        l += p[kb][r];
      }

    // O^T += V^T P^T. Operand element t of k-step st2 (lane half hi) is key
    // 16*st2 + 8*(t/4) + 4*hi + t%4, which the transposed tile stores as 8 consecutive
    // elements at position 16*st2 + 8*hi.
#pragma unroll
    for (int kb = 0; kb < kBN / 32; ++kb) {
#pragma unroll
      for (int st2 = 0; st2 < 2; ++st2) {
        const bf16x8 pb = to_bf16x8(&p[kb][8 * st2]);
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          const bf16x8 af = *(const VC_LDS bf16x8*)(vt_lds + ((db * 32 + l32) * kTileRow + kb * 32 + 16 * st2 + 8 * hi) * 2);
          oacc[db] = mfma32(af, pb, oacc[db]);
        }
      }
    }
    st ^= 1;
    kt = kn;
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
    hipLaunchKernelGGL(fwd_kernel<128>, grid, dim3(64 * kWaves), 0, s, a);
  else
    hipLaunchKernelGGL(fwd_kernel<64>, grid, dim3(64 * kWaves), 0, s, a);
  return hipGetLastError();
}

}  // namespace vcja
