// Temporal attention branch for gfx950: each spatial position attends across the
// frames (the [B*L, F, ...] regrouping of the multimodal diffusion block), read in
// place from the joint [B, N, H, D] layout where video token (f, l) is row T + f*L + l.
//
// Sequences are short (F <= 32), so one wave packs G = floor(32/F) consecutive
// positions of one (sample, head) into the 32 slots of a 32x32x16 matrix-core
// block: slot s holds frame s % F of position l0 + s / F; slots past G*F are
// padding. Rows of Q, K (and dO, V in the backward) are read as 16-byte chunks, one
// slot per lane; the rows whose transposes are MFMA operands (V^T in the forward,
// K^T, Q^T, dO^T in the backward) are also written to LDS, and the transposed
// fragments read from there element by element in the key order the accumulator
// layout produces. A key is valid for a query if it belongs to the
// same position (same group of F slots) and key_mask keeps it. The work is small
// and bound by memory traffic.
#include "common.hpp"

namespace vcja {
namespace {

constexpr int kSlots = 32;
constexpr int kWavesPerBlock = 4;
// Rows of a wave's 32 slots staged in LDS (row-major, padded by 8 elements so that the
// rows of a 16-byte write fall in different banks): transposed operands are read from
// there two bytes at a time instead of being gathered from memory.
constexpr int kRowPad = 8;
template <int D>
constexpr int stage_elems() { return kSlots * (D + kRowPad); }

// Token row of slot s in the block starting at position l0 (clamped into range for
// padding slots, whose probabilities are zero).
struct SlotMap {
  int T, F, L, G, l0;
  __device__ __forceinline__ bool ok(int s) const { return s < G * F && l0 + s / F < L; }
  __device__ __forceinline__ int token(int s) const {
    const int g = s / F;
    const int f = s - g * F;
    const int l = l0 + g < L ? l0 + g : l0;
    return T + f * L + l;
  }
};

// Slot held by register r of a lane of half hi in a 32x32 accumulator (row index).
__device__ __forceinline__ int acc_slot(int r, int hi) { return acc_row(r, hi); }

// Slot of operand element t of k-step st for a lane of half hi: the order in which the
// accumulator rows of 8 consecutive registers are numbered.
__device__ __forceinline__ int op_slot(int st, int t, int hi) { return 16 * st + 8 * (t >> 2) + 4 * hi + (t & 3); }

// Sum of three bf16 values in fp32, in argument order, rounded once (a NULL source counts as
// zero): the arithmetic shared by the branch-sum kernel and the fused epilogue.
__device__ __forceinline__ void add_bf16x4(f32x4& acc, bf16x4 x) {
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] += (float)x[i];
}
__device__ __forceinline__ void add_bf16x4(f32x4& acc, const __bf16* src) {
  if (src) add_bf16x4(acc, *(const bf16x4*)src);
}
__device__ __forceinline__ void add_bf16x8(f32x4& lo, f32x4& hi, bf16x8 x) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    lo[i] += (float)x[i];
    hi[i] += (float)x[4 + i];
  }
}

// One wave: attention of the G positions starting at sm.l0 (sm.l0 < L) of head h, sample b.
template <int D>
__device__ __forceinline__ void temporal_fwd_wave(const TemporalArgs& a, const SlotMap& sm, int h, int b,
                                                  VC_LDS __bf16* vs) {
  const int lane = threadIdx.x & 63;
  const int l32 = lane & 31;
  const int hi = lane >> 5;
  const size_t tok = (size_t)a.H * D;
  const size_t base = (size_t)b * a.N * tok + (size_t)h * D;

  // This lane's slot as query (B operand column) and as key (A operand row).
  const int s = l32;
  const int g = s / a.F;
  const bool q_ok = sm.ok(s);
  const int n = sm.token(s);
  bf16x8 qf[D / 16], kf[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    qf[ks] = *(const bf16x8*)(a.q + base + (size_t)n * tok + 16 * ks + 8 * hi);
    kf[ks] = *(const bf16x8*)(a.k + base + (size_t)n * tok + 16 * ks + 8 * hi);
    *(VC_LDS bf16x8*)(vs + s * (D + kRowPad) + 16 * ks + 8 * hi) =
        *(const bf16x8*)(a.v + base + (size_t)n * tok + 16 * ks + 8 * hi);
  }
  // S^T = K Q^T: lane column = query slot s, register r = key slot acc_slot(r, hi).
  f32x16 sacc = zero_f32x16();
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) sacc = mfma32(kf[ks], qf[ks], sacc);

  // Keys of the same group (position) only; padding and masked keys excluded.
  const int lo = g * a.F;
  const uint8_t* km = a.key_mask ? a.key_mask + (size_t)b * a.N : nullptr;
  float mx = -INFINITY;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int j = acc_slot(r, hi);
    bool ok = q_ok & (j >= lo) & (j < lo + a.F);
    if (km) ok = ok & (km[sm.token(j)] != 0);
    sacc[r] = ok ? sacc[r] : -INFINITY;
    mx = fmaxf(mx, sacc[r]);
  }
  mx = halves_max(mx);
  const float m2 = mx == -INFINITY ? 0.0f : mx * a.scale_log2;
  float p[16], sum = 0.0f;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    p[r] = fast_exp2(fmaf(sacc[r], a.scale_log2, -m2));
    sum += p[r];
  }
  sum = halves_sum(sum);

  // O^T = V^T P^T over the 32 key slots (two k-steps of 16).
  bf16x8 pb[2];
  pb[0] = to_bf16x8(&p[0]);
  pb[1] = to_bf16x8(&p[8]);
  int vrow[2][8];  // LDS rows of the key slots of operand element t, k-step st
#pragma unroll
  for (int st = 0; st < 2; ++st)
#pragma unroll
    for (int t = 0; t < 8; ++t) vrow[st][t] = op_slot(st, t, hi) * (D + kRowPad);
  const float inv = sum > 0.0f ? 1.0f / sum : 0.0f;
  __bf16* op = a.o + base + (size_t)n * tok;
#pragma unroll
  for (int db = 0; db < D / 32; ++db) {
    f32x16 oacc = zero_f32x16();
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      bf16x8 vt;
#pragma unroll
      for (int t = 0; t < 8; ++t) vt[t] = vs[vrow[st][t] + db * 32 + l32];
      oacc = mfma32(vt, pb[st], oacc);
    }
    if (q_ok) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        bf16x4 o4 = {(__bf16)(oacc[4 * j + 0] * inv), (__bf16)(oacc[4 * j + 1] * inv),
                     (__bf16)(oacc[4 * j + 2] * inv), (__bf16)(oacc[4 * j + 3] * inv)};
        *(bf16x4*)(op + db * 32 + 8 * j + 4 * hi) = o4;
      }
    }
  }
  if (q_ok && hi == 0)
    a.lse[((size_t)b * a.H + h) * a.N + n] = sum > 0.0f ? (m2 + __log2f(sum)) * kLn2 : -INFINITY;
}

// Forward: one wave per G positions. With SUM, the workgroup then writes the branch sum
// sum_out = (sum_a + sum_b) + o of the rows it produced, reading o back after a barrier
// so that every access is a whole 16-byte chunk of a row (the accumulator layout would
// scatter 8-byte pieces over 32 rows per instruction).
template <int D, bool SUM>
__global__ __launch_bounds__(64 * kWavesPerBlock) void temporal_fwd_kernel(TemporalArgs a) {
  const int h = blockIdx.y;
  const int b = blockIdx.z;
  __shared__ __attribute__((aligned(16))) __bf16 stage[kWavesPerBlock * stage_elems<D>()];
  const int wave = threadIdx.x >> 6;
  SlotMap sm{a.T, a.F, a.L, a.G, (int)(blockIdx.x * kWavesPerBlock + wave) * a.G};
  if (sm.l0 < a.L) temporal_fwd_wave<D>(a, sm, h, b, (VC_LDS __bf16*)stage + wave * stage_elems<D>());
  if (SUM) {
    __syncthreads();  // this workgroup's rows of o are written
    const int wl0 = (int)blockIdx.x * kWavesPerBlock * a.G;  // first position of the workgroup
    const int npos = min(kWavesPerBlock * a.G, a.L - wl0);
    constexpr int kChunks = D / 8;  // 16-byte chunks per row
    const size_t tok = (size_t)a.H * D;
    const size_t base = (size_t)b * a.N * tok + (size_t)h * D;
    for (int i = threadIdx.x; i < a.F * npos * kChunks; i += blockDim.x) {
      const int r = i / kChunks;
      const int f = r / npos;
      const size_t off = base + (size_t)(a.T + f * a.L + wl0 + (r - f * npos)) * tok + (i % kChunks) * 8;
      f32x4 lo = {0.0f, 0.0f, 0.0f, 0.0f}, hi = lo;
      if (a.sum_a) add_bf16x8(lo, hi, *(const bf16x8*)(a.sum_a + off));
      if (a.sum_b) add_bf16x8(lo, hi, *(const bf16x8*)(a.sum_b + off));
      add_bf16x8(lo, hi, *(const bf16x8*)(a.o + off));
      bf16x8 r8;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        r8[e] = (__bf16)lo[e];
        r8[4 + e] = (__bf16)hi[e];
      }
      *(bf16x8*)(a.sum_out + off) = r8;
    }
  }
}

// Backward. LSE*log2(e) and -D = -rowsum(dO o O) per token come from the preparation pass
// ([B, H, npad], +inf / 0 where a row has no key). Two orientations of the same block:
// lane = query (S^T, dP^T, dS^T) gives dQ^T = c K^T dS^T; lane = key (S, dP, dS) gives
// dV^T = dO^T P and dK^T = c Q^T dS. The transposed A operands are gathered in the slot
// order the accumulator layout produces.
template <int D>
__global__ __launch_bounds__(64 * kWavesPerBlock) void temporal_bwd_kernel(TemporalArgs a) {
  // Per wave: K rows of its 32 slots (the dQ part), later Q rows in the same place (the
  // dK/dV part), dO rows; then LSE*log2e and -D of the slots. Two workgroups fit a CU.
  __shared__ __attribute__((aligned(16))) __bf16 stage[kWavesPerBlock * 2 * stage_elems<D>()];
  __shared__ float stat[kWavesPerBlock * 2 * kSlots];
  const int lane = threadIdx.x & 63;
  const int l32 = lane & 31;
  const int hi = lane >> 5;
  const int wave = threadIdx.x >> 6;
  VC_LDS __bf16* k_rows = (VC_LDS __bf16*)stage + wave * 2 * stage_elems<D>();
  VC_LDS __bf16* q_rows = k_rows;  // once the dQ part has read K
  VC_LDS __bf16* do_rows = k_rows + stage_elems<D>();
  VC_LDS float* lse_slot = (VC_LDS float*)stat + wave * 2 * kSlots;
  VC_LDS float* nd_slot = lse_slot + kSlots;
  const int blk = blockIdx.x * kWavesPerBlock + wave;
  const int h = blockIdx.y;
  const int b = blockIdx.z;
  SlotMap sm{a.T, a.F, a.L, a.G, blk * a.G};
  if (sm.l0 >= a.L) return;  // whole wave
  const size_t tok = (size_t)a.H * D;
  const size_t base = (size_t)b * a.N * tok + (size_t)h * D;
  const uint8_t* km = a.key_mask ? a.key_mask + (size_t)b * a.N : nullptr;

  const int s = l32;  // this lane's slot (query in one orientation, key in the other)
  const int lo = (s / a.F) * a.F;
  const bool s_ok = sm.ok(s);
  const int n = sm.token(s);
  bf16x8 qf[D / 16], kf[D / 16], vf[D / 16], dof[D / 16];
  float dsum = 0.0f;  // this half's share of D = <dO, O> of the slot's token
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    const size_t off = base + (size_t)n * tok + 16 * ks + 8 * hi;
    qf[ks] = *(const bf16x8*)(a.q + off);
    kf[ks] = *(const bf16x8*)(a.k + off);
    vf[ks] = *(const bf16x8*)(a.v + off);
    dof[ks] = *(const bf16x8*)(a.dout + off);
    const bf16x8 of = *(const bf16x8*)(a.o_in + off);
#pragma unroll
    for (int e = 0; e < 8; ++e) dsum = fmaf((float)dof[ks][e], (float)of[e], dsum);
    const int e = s * (D + kRowPad) + 16 * ks + 8 * hi;
    *(VC_LDS bf16x8*)(k_rows + e) = kf[ks];
    *(VC_LDS bf16x8*)(do_rows + e) = dof[ks];
  }
  // -D and LSE*log2(e) of the slot's token, formed here from O and the forward's LSE (no
  // preparation pass): LSE*log2(e) is +inf where the token has no valid key or the slot
  // none, so that its probabilities vanish.
  const float lse_n = a.lse[((size_t)b * a.H + h) * a.N + n];
  const float l2 = (s_ok && lse_n != -INFINITY) ? lse_n * kLog2e : INFINITY;
  const float d = s_ok ? -halves_sum(dsum) : 0.0f;
  if (hi == 0) {
    lse_slot[s] = l2;
    nd_slot[s] = d;
  }
  // LDS rows of the slots an operand element t of k-step st refers to.
  int grow[2][8];
#pragma unroll
  for (int st = 0; st < 2; ++st)
#pragma unroll
    for (int t = 0; t < 8; ++t) grow[st][t] = op_slot(st, t, hi) * (D + kRowPad);

  // ---- lane = query: dQ ----
  {
    f32x16 sacc = zero_f32x16(), pacc = zero_f32x16();
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      sacc = mfma32(kf[ks], qf[ks], sacc);
      pacc = mfma32(vf[ks], dof[ks], pacc);
    }
    float ds[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int j = acc_slot(r, hi);
      bool ok = s_ok & (j >= lo) & (j < lo + a.F);
      if (km) ok = ok & (km[sm.token(j)] != 0);
      const float p = ok ? fast_exp2(fmaf(sacc[r], a.scale_log2, -l2)) : 0.0f;
      ds[r] = p * (pacc[r] + d);
    }
    bf16x8 sb[2];
    sb[0] = to_bf16x8(&ds[0]);
    sb[1] = to_bf16x8(&ds[8]);
    __bf16* dqp = a.o + base + (size_t)n * tok;
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      f32x16 acc = zero_f32x16();
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        bf16x8 kt;
#pragma unroll
        for (int t = 0; t < 8; ++t) kt[t] = k_rows[grow[st][t] + db * 32 + l32];
        acc = mfma32(kt, sb[st], acc);
      }
      if (s_ok) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          bf16x4 o4 = {(__bf16)(acc[4 * j + 0] * a.scale), (__bf16)(acc[4 * j + 1] * a.scale),
                       (__bf16)(acc[4 * j + 2] * a.scale), (__bf16)(acc[4 * j + 3] * a.scale)};
          *(bf16x4*)(dqp + db * 32 + 8 * j + 4 * hi) = o4;
        }
      }
    }
  }
  // ---- lane = key: dK, dV ----
  // Q rows replace the K rows (LDS operations of a wave complete in order, so every read
  // of K above precedes these writes).
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) *(VC_LDS bf16x8*)(q_rows + s * (D + kRowPad) + 16 * ks + 8 * hi) = qf[ks];
  {
    f32x16 sacc = zero_f32x16(), pacc = zero_f32x16();
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      sacc = mfma32(qf[ks], kf[ks], sacc);
      pacc = mfma32(dof[ks], vf[ks], pacc);
    }
    bool k_ok = s_ok;
    if (km) k_ok = k_ok & (km[n] != 0);
    float p[16], ds[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = acc_slot(r, hi);  // query slot
      const bool ok = k_ok & (i >= lo) & (i < lo + a.F) & sm.ok(i);
      const float l2 = lse_slot[i];
      const float d = nd_slot[i];
      p[r] = ok ? fast_exp2(fmaf(sacc[r], a.scale_log2, -l2)) : 0.0f;
      ds[r] = p[r] * (pacc[r] + d);
    }
    bf16x8 pb[2], sb[2];
    pb[0] = to_bf16x8(&p[0]);
    pb[1] = to_bf16x8(&p[8]);
    sb[0] = to_bf16x8(&ds[0]);
    sb[1] = to_bf16x8(&ds[8]);
    __bf16* dkp = a.dk + base + (size_t)n * tok;
    __bf16* dvp = a.dv + base + (size_t)n * tok;
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      f32x16 vacc = zero_f32x16(), kacc = zero_f32x16();
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        bf16x8 dot, qt;
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          dot[t] = do_rows[grow[st][t] + db * 32 + l32];
          qt[t] = q_rows[grow[st][t] + db * 32 + l32];
        }
        vacc = mfma32(dot, pb[st], vacc);
        kacc = mfma32(qt, sb[st], kacc);
      }
      if (s_ok) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          bf16x4 v4 = {(__bf16)vacc[4 * j + 0], (__bf16)vacc[4 * j + 1], (__bf16)vacc[4 * j + 2],
                       (__bf16)vacc[4 * j + 3]};
          bf16x4 k4 = {(__bf16)(kacc[4 * j + 0] * a.scale), (__bf16)(kacc[4 * j + 1] * a.scale),
                       (__bf16)(kacc[4 * j + 2] * a.scale), (__bf16)(kacc[4 * j + 3] * a.scale)};
          *(bf16x4*)(dvp + db * 32 + 8 * j + 4 * hi) = v4;
          *(bf16x4*)(dkp + db * 32 + 8 * j + 4 * hi) = k4;
        }
      }
    }
  }
}

// out = a + b + c (fp32, in that order, one rounding) over rows [0, rows) of each sample;
// one thread per 4 elements.
__global__ __launch_bounds__(256) void branch_sum_kernel(const __bf16* a, const __bf16* b, const __bf16* c,
                                                         __bf16* out, int B, int N, int rows, int row_elems) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int per_row = row_elems / 4;
  if (i >= (size_t)B * rows * per_row) return;
  const size_t r = i / per_row;
  const size_t off = ((r / rows) * N + r % rows) * row_elems + (i % per_row) * 4;
  f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  add_bf16x4(acc, a ? a + off : nullptr);
  add_bf16x4(acc, b ? b + off : nullptr);
  add_bf16x4(acc, c ? c + off : nullptr);
  *(bf16x4*)(out + off) = bf16x4{(__bf16)acc[0], (__bf16)acc[1], (__bf16)acc[2], (__bf16)acc[3]};
}

// Zero rows [0, T) of up to three tensors and set their LSE to -inf.
template <int D>
__global__ __launch_bounds__(256) void text_rows_kernel(__bf16* x0, __bf16* x1, __bf16* x2, float* lse, int B, int H,
                                                        int N, int T) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;  // one 16-byte chunk
  constexpr int CPR = D / 8;
  const size_t rows = (size_t)B * T * H;
  if (i < rows * CPR) {
    const size_t row = i / CPR;
    const int c = (int)(i % CPR);
    const int hh = (int)(row % H);
    const size_t bt = row / H;
    const int t = (int)(bt % T);
    const int b = (int)(bt / T);
    const size_t off = (((size_t)b * N + t) * H + hh) * D + c * 8;
    const bf16x8 z = zero_bf16x8();
    if (x0) *(bf16x8*)(x0 + off) = z;
    if (x1) *(bf16x8*)(x1 + off) = z;
    if (x2) *(bf16x8*)(x2 + off) = z;
    if (lse && c == 0) lse[((size_t)b * H + hh) * N + t] = -INFINITY;
  }
}

}  // namespace

hipError_t launch_temporal_fwd(const TemporalArgs& a, int head_dim, hipStream_t s) {
  const int nblk = (a.L + a.G - 1) / a.G;
  dim3 grid((nblk + kWavesPerBlock - 1) / kWavesPerBlock, a.H, a.B);
  const bool sum = a.sum_out != nullptr;
  if (head_dim == 128 && sum)
    hipLaunchKernelGGL((temporal_fwd_kernel<128, true>), grid, dim3(64 * kWavesPerBlock), 0, s, a);
  else if (head_dim == 128)
    hipLaunchKernelGGL((temporal_fwd_kernel<128, false>), grid, dim3(64 * kWavesPerBlock), 0, s, a);
  else if (sum)
    hipLaunchKernelGGL((temporal_fwd_kernel<64, true>), grid, dim3(64 * kWavesPerBlock), 0, s, a);
  else
    hipLaunchKernelGGL((temporal_fwd_kernel<64, false>), grid, dim3(64 * kWavesPerBlock), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_branch_sum(const __bf16* a, const __bf16* b, const __bf16* c, __bf16* out, int B, int N, int rows,
                             int row_elems, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const size_t threads = (size_t)B * rows * (row_elems / 4);
  hipLaunchKernelGGL(branch_sum_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, a, b, c, out, B, N,
                     rows, row_elems);
  return hipGetLastError();
}

hipError_t launch_temporal_bwd(const TemporalArgs& a, int head_dim, hipStream_t s) {
  const int nblk = (a.L + a.G - 1) / a.G;
  dim3 grid((nblk + kWavesPerBlock - 1) / kWavesPerBlock, a.H, a.B);
  if (head_dim == 128)
    hipLaunchKernelGGL(temporal_bwd_kernel<128>, grid, dim3(64 * kWavesPerBlock), 0, s, a);
  else
    hipLaunchKernelGGL(temporal_bwd_kernel<64>, grid, dim3(64 * kWavesPerBlock), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_text_rows(__bf16* x0, __bf16* x1, __bf16* x2, float* lse, int B, int H, int N, int T, int head_dim,
                            hipStream_t s) {
  if (T <= 0) return hipSuccess;
  const size_t chunks = (size_t)B * T * H * (head_dim / 8);
  dim3 grid((unsigned)((chunks + 255) / 256));
  if (head_dim == 128)
    hipLaunchKernelGGL(text_rows_kernel<128>, grid, dim3(256), 0, s, x0, x1, x2, lse, B, H, N, T);
  else
    hipLaunchKernelGGL(text_rows_kernel<64>, grid, dim3(256), 0, s, x0, x1, x2, lse, B, H, N, T);
  return hipGetLastError();
}

}  // namespace vcja
