// Temporal attention branch for gfx950: each spatial position attends across the
// frames (the [B*L, F, ...] regrouping of the multimodal diffusion block), read in
// place from the joint [B, N, H, D] layout where video token (f, l) is row T + f*L + l.
//
// Sequences are short (F <= 32), so one workgroup packs G = floor(32/F) consecutive
// positions of one (sample, head) into the 32 slots of a 32x32x16 matrix-core block:
// slot s holds frame s % F of position l0 + s / F; slots past G*F are padding. The
// rows of the slots are copied into LDS row tiles by whole-row wave copies (64 lanes
// read consecutive 16-byte chunks of a few token rows: one slot per lane would make
// every lane's chunk its own cache access), the MFMA operands are read from there
// (transposing reads where the contraction runs over slots), and the results go back
// through a tile so that they too are stored as whole rows. A key is valid for a query
// if it belongs to the same position (same group of F slots) and key_mask keeps it. The
// work is small and bound by memory traffic.
#include "common.hpp"

namespace vcja {
namespace {

constexpr int kSlots = 32;

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

// Row tiles of a group's 32 slots in LDS: slot s sits in row perm_row(s)
// (the permuted order of the joint backward, so that the transposing reads of four
// consecutive slots hit distinct banks) with one 16-byte pad chunk per row (the rows one
// quarter-wave reads at a common column fall on distinct banks), filled by whole 1 KiB wave
// copies in which 64 lanes read consecutive 16-byte chunks of a few token rows.
template <int D>
struct SlotTile {
  static constexpr int CH = D / 8 + 1;                     // 16-byte chunks per row, pad included
  static constexpr int RS = CH * 16;                       // row stride (bytes)
  static constexpr int COPIES = (kSlots * CH + 63) / 64;   // wave copies per tensor
  static constexpr int REGION = COPIES * 1024;             // LDS bytes per tensor
};

// Issues wave copy `idx` of the 32 slot rows of one tensor (token row n at src + n*tok) into
// `dst`. `tk` holds the token row of slot l32 in lane l32. Lanes past the last row repeat
// one of its chunks (their bytes land in the region's tail, which nothing reads); the pad
// chunk of a row repeats the row's last chunk.
template <int D>
__device__ __forceinline__ void copy_slot_rows(const __bf16* src, size_t tok, int tk, VC_LDS char* dst, int idx,
                                               int lane) {
  constexpr int CH = SlotTile<D>::CH;
  const int lin = idx * 64 + lane;
  const int r = lin / CH;
  const int c = min(lin - r * CH, CH - 2);
  const int n = __shfl(tk, perm_row(min(r, kSlots - 1)));
  copy16_to_lds_opaque(src + (size_t)n * tok + c * 8, dst + idx * 1024);
}

// MFMA operand from slot rows (m = slot l32, k = dims 16*ks + 8*hi .. +7).
template <int D>
__device__ __forceinline__ bf16x8 slot_rows(const VC_LDS char* t, int ks, int lane) {
  return *(const VC_LDS bf16x8*)(t + perm_row(lane & 31) * SlotTile<D>::RS + (2 * ks + (lane >> 5)) * 16);
}

// MFMA operand whose contraction runs over slots (m = dim db*32 + l32, k = slots
// 16*st + 8*(t/4) + 4*hi + t%4, the order an accumulator column holds them): two transposing
// reads of 4 slots each; lane 4e+g of a group of 16 supplies the address of slot r0 + e and
// 4 dims.
template <int D>
__device__ __forceinline__ bf16x8 slot_cols(const VC_LDS char* t, int st, int db, int lane) {
  const int e = (lane & 15) >> 2;
  const int col = (db * 32 + 16 * ((lane >> 4) & 1) + 4 * (lane & 3)) * 2;
  const int r0 = 16 * st + 4 * (lane >> 5) + e;
  const bf16x4 x = lds_read_tr(t + perm_row(r0) * SlotTile<D>::RS + col);
  const bf16x4 y = lds_read_tr(t + perm_row(r0 + 8) * SlotTile<D>::RS + col);
  return cat4(x, y);
}

// Forward: one wave per group of G positions (32 slots) of one (sample, head), head fastest
// over the grid, so that concurrent workgroups read whole token rows. Q, K and V rows are
// copied into LDS row tiles; lane = query: S^T = K Q^T, the softmax over the lane's group
// with fp32 sums, O^T = V^T P^T (P rounded to bf16 for the product). O goes back through
// the Q tile so that it is stored as whole rows; with SUM the same rows of the branch sum
// sum_out = (sum_a + sum_b) + o are formed from them and written too.
template <int D, bool SUM>
__global__ __launch_bounds__(64) void temporal_fwd_kernel(TemporalArgs a) {
  using Tile = SlotTile<D>;
  constexpr int LPR = D / 8;     // lanes per row in a whole-row access
  constexpr int RPI = 64 / LPR;  // rows per whole-row wave access
  constexpr int NR = kSlots / RPI;
  __shared__ __attribute__((aligned(1024))) char smem[3 * Tile::REGION];
  VC_LDS char* const q_t = (VC_LDS char*)smem;
  VC_LDS char* const k_t = q_t + Tile::REGION;
  VC_LDS char* const v_t = k_t + Tile::REGION;

  const int lane = threadIdx.x & 63;
  const int l32 = lane & 31;
  const int hi = lane >> 5;
  const int nblk = (a.L + a.G - 1) / a.G;
  const int h = (int)(blockIdx.x % a.H);
  const int pb = (int)(blockIdx.x / a.H) % nblk;
  const int b = (int)(blockIdx.x / a.H) / nblk;
  const SlotMap sm{a.T, a.F, a.L, a.G, pb * a.G};
  const size_t tok = (size_t)a.H * D;
  const size_t base = (size_t)b * a.N * tok + (size_t)h * D;
  const int tk = sm.token(l32);  // token row of slot l32 (lanes l32 and l32 + 32 alike)
  const unsigned vbits = (unsigned)__ballot(sm.ok(l32));  // valid slots
  const int ch = lane % LPR;
#pragma unroll
  for (int idx = 0; idx < Tile::COPIES; ++idx) {
    copy_slot_rows<D>(a.q + base, tok, tk, q_t, idx, lane);
    copy_slot_rows<D>(a.k + base, tok, tk, k_t, idx, lane);
    copy_slot_rows<D>(a.v + base, tok, tk, v_t, idx, lane);
  }
  // With SUM, the rows of the other two branch outputs this lane adds, as whole-row loads
  // (from q in place of a missing one: any readable bytes, replaced by zero below).
  bf16x8 ra[SUM ? NR : 1], rb[SUM ? NR : 1];
  if constexpr (SUM) {
#pragma unroll
    for (int i = 0; i < NR; ++i) {
      const size_t off = base + (size_t)__shfl(tk, RPI * i + lane / LPR) * tok + ch * 8;
      ra[i] = *(const bf16x8*)((a.sum_a ? a.sum_a : a.q) + off);
      rb[i] = *(const bf16x8*)((a.sum_b ? a.sum_b : a.q) + off);
    }
  }
  // Key-mask byte of slot l32, loaded unconditionally (from any readable byte if there is no
  // mask) so that no branch waits for it among the copies.
  int kmb = *(a.key_mask ? a.key_mask + (size_t)b * a.N + tk : (const uint8_t*)a.q);
  // Every load above is used only after this full wait (one wave: its copies are then in
  // LDS); a wait for any one of them would wait for the copies issued before it too.
  wait_all_memory();
  asm volatile("" : "+v"(kmb));  // the mask test stays after the wait
  const unsigned kbits = (unsigned)__ballot(!a.key_mask || kmb != 0) & vbits;  // valid, unmasked keys

  // lane = query l32; register r = key acc_row(r, hi). Keys of the query's own position
  // (its group of F slots) only.
  const int lo = (l32 / a.F) * a.F;
  const unsigned group = a.F == kSlots ? ~0u : ((1u << a.F) - 1u) << lo;
  const bool q_ok = (vbits >> l32) & 1;
  const unsigned allow = (q_ok ? group & kbits : 0u) >> (4 * hi);
  f32x16 sacc = zero_f32x16();
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) sacc = mfma32(slot_rows<D>(k_t, ks, lane), slot_rows<D>(q_t, ks, lane), sacc);
  float mx = -INFINITY;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const bool ok = (allow >> (8 * (r >> 2) + (r & 3))) & 1;
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
  const bf16x8 pb0 = to_bf16x8(&p[0]), pb1 = to_bf16x8(&p[8]);
  const float inv = sum > 0.0f ? 1.0f / sum : 0.0f;
  bf16x4 res[D / 32][4];
#pragma unroll
  for (int db = 0; db < D / 32; ++db) {
    f32x16 oacc = zero_f32x16();
    oacc = mfma32(slot_cols<D>(v_t, 0, db, lane), pb0, oacc);
    oacc = mfma32(slot_cols<D>(v_t, 1, db, lane), pb1, oacc);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      res[db][j] = bf16x4{(__bf16)(oacc[4 * j] * inv), (__bf16)(oacc[4 * j + 1] * inv),
                          (__bf16)(oacc[4 * j + 2] * inv), (__bf16)(oacc[4 * j + 3] * inv)};
  }
  if (q_ok && hi == 0)
    a.lse[((size_t)b * a.H + h) * a.N + tk] = sum > 0.0f ? (m2 + __log2f(sum)) * kLn2 : -INFINITY;
  // O rows through the Q tile (every read of it above precedes these writes: LDS operations
  // of a wave complete in order), then whole-row stores of the valid slots.
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      *(VC_LDS bf16x4*)(q_t + perm_row(l32) * Tile::RS + (db * 32 + 8 * j + 4 * hi) * 2) = res[db][j];
#pragma unroll
  for (int i = 0; i < NR; ++i) {
    const int sl = RPI * i + lane / LPR;
    const size_t off = base + (size_t)__shfl(tk, sl) * tok + ch * 8;
    const bf16x8 row = *(const VC_LDS bf16x8*)(q_t + perm_row(sl) * Tile::RS + ch * 16);
    if ((vbits >> sl) & 1) {
      *(bf16x8*)(a.o + off) = row;
      if constexpr (SUM) {
        f32x4 lo4 = {0.0f, 0.0f, 0.0f, 0.0f}, hi4 = lo4;
        add_bf16x8(lo4, hi4, a.sum_a ? ra[i] : zero_bf16x8());
        add_bf16x8(lo4, hi4, a.sum_b ? rb[i] : zero_bf16x8());
        add_bf16x8(lo4, hi4, row);
        bf16x8 r8;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          r8[e] = (__bf16)lo4[e];
          r8[4 + e] = (__bf16)hi4[e];
        }
        *(bf16x8*)(a.sum_out + off) = r8;
      }
    }
  }
}

// Backward: one workgroup of two waves per group of G positions (32 slots) of one (sample,
// head), head fastest over the grid, so that concurrent workgroups read whole token rows.
// Q, K, V and dO rows are copied into LDS row tiles by whole-row wave copies; D = <dO, O>
// (O read as whole rows) and LSE*log2(e) of every slot are formed first and shared through
// LDS. Wave 0 takes the lane-per-query orientation (S^T = K Q^T, dP^T = V dO^T, dS^T) and
// forms dQ^T = c K^T dS^T; wave 1 the lane-per-key one (S, dP, dS) and forms dV^T = dO^T P
// and dK^T = c Q^T dS. The results go back through the tiles so that every global store is
// a whole 16-byte chunk of a row.
template <int D>
__global__ __launch_bounds__(128) void temporal_bwd_kernel(TemporalArgs a) {
  using Tile = SlotTile<D>;
  constexpr int LPR = D / 8;   // lanes per row in a whole-row access
  constexpr int RPI = 64 / LPR;  // rows per whole-row wave access
  __shared__ __attribute__((aligned(1024))) char smem[4 * Tile::REGION + 2 * kSlots * 4];
  VC_LDS char* const q_t = (VC_LDS char*)smem;
  VC_LDS char* const k_t = q_t + Tile::REGION;
  VC_LDS char* const v_t = k_t + Tile::REGION;
  VC_LDS char* const do_t = v_t + Tile::REGION;
  VC_LDS float* const lse_slot = (VC_LDS float*)(do_t + Tile::REGION);  // LSE*log2(e), +inf if none
  VC_LDS float* const nd_slot = lse_slot + kSlots;                      // -D, 0 if none

  const int lane = threadIdx.x & 63;
  const int l32 = lane & 31;
  const int hi = lane >> 5;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nblk = (a.L + a.G - 1) / a.G;
  const int h = (int)(blockIdx.x % a.H);
  const int pb = (int)(blockIdx.x / a.H) % nblk;
  const int b = (int)(blockIdx.x / a.H) / nblk;
  const SlotMap sm{a.T, a.F, a.L, a.G, pb * a.G};
  const size_t tok = (size_t)a.H * D;
  const size_t base = (size_t)b * a.N * tok + (size_t)h * D;
  const int tk = sm.token(l32);  // token row of slot l32 (lanes l32 and l32 + 32 alike)
  const unsigned vbits = (unsigned)__ballot(sm.ok(l32));  // valid slots

  // Row copies: wave 0 Q and K, wave 1 V and dO.
  {
    const __bf16* s0 = (w == 0 ? a.q : a.v) + base;
    const __bf16* s1 = (w == 0 ? a.k : a.dout) + base;
    VC_LDS char* d0 = w == 0 ? q_t : v_t;
    VC_LDS char* d1 = w == 0 ? k_t : do_t;
#pragma unroll
    for (int idx = 0; idx < Tile::COPIES; ++idx) {
      copy_slot_rows<D>(s0, tok, tk, d0, idx, lane);
      copy_slot_rows<D>(s1, tok, tk, d1, idx, lane);
    }
  }
  // This wave's 16 slots of D = <dO, O>: O rows as whole-row loads.
  constexpr int NI = 16 / RPI;
  const int ch = lane % LPR;
  bf16x8 of[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int n = __shfl(tk, 16 * w + RPI * i + lane / LPR);
    of[i] = *(const bf16x8*)(a.o_in + base + (size_t)n * tok + ch * 8);
  }
  const int n16 = __shfl(tk, 16 * w + (lane & 15));
  const float lse_v = a.lse[((size_t)b * a.H + h) * a.N + n16];
  // Key-mask byte of slot l32, loaded unconditionally (from any readable byte if there is no
  // mask) so that no branch waits for it among the copies.
  int kmb = *(a.key_mask ? a.key_mask + (size_t)b * a.N + tk : (const uint8_t*)a.lse);
  // Every load above is used only after this full wait: a wait for any one of them would
  // wait for the row copies issued before it too.
  wait_all_memory();
  asm volatile("" : "+v"(kmb));  // the mask test stays after the wait
  __syncthreads();               // every row copy has landed
  const unsigned kbits = (unsigned)__ballot(!a.key_mask || kmb != 0) & vbits;  // valid, unmasked keys
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int sl = 16 * w + RPI * i + lane / LPR;
    const bf16x8 dv = *(const VC_LDS bf16x8*)(do_t + perm_row(sl) * Tile::RS + ch * 16);
    float acc = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = fmaf((float)dv[e], (float)of[i][e], acc);
#pragma unroll
    for (int m = 1; m < LPR; m <<= 1) acc += __shfl_xor(acc, m);
    if (ch == 0) nd_slot[sl] = (vbits >> sl) & 1 ? -acc : 0.0f;
  }
  if (lane < 16) {
    const int sl = 16 * w + lane;
    lse_slot[sl] = ((vbits >> sl) & 1) && lse_v != -INFINITY ? lse_v * kLog2e : INFINITY;
  }
  __syncthreads();  // statistics of every slot are in LDS

  // Slots of this lane's group (the position of slot l32): [lo, lo + F).
  const int lo = (l32 / a.F) * a.F;
  const unsigned group = a.F == kSlots ? ~0u : ((1u << a.F) - 1u) << lo;
  bf16x4 res[2][D / 32][4];  // wave 0: dQ^T in res[0]; wave 1: dV^T in res[0], dK^T in res[1]
  if (w == 0) {
    // lane = query l32; register r = key acc_row(r, hi)
    f32x16 sacc = zero_f32x16(), pacc = zero_f32x16();
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      sacc = mfma32(slot_rows<D>(k_t, ks, lane), slot_rows<D>(q_t, ks, lane), sacc);
      pacc = mfma32(slot_rows<D>(v_t, ks, lane), slot_rows<D>(do_t, ks, lane), pacc);
    }
    const unsigned allow = (((vbits >> l32) & 1) ? group & kbits : 0u) >> (4 * hi);
    const float l2 = lse_slot[l32];
    const float d = nd_slot[l32];
    float ds[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const bool ok = (allow >> (8 * (r >> 2) + (r & 3))) & 1;
      const float p = ok ? fast_exp2(fmaf(sacc[r], a.scale_log2, -l2)) : 0.0f;
      ds[r] = p * (pacc[r] + d);
    }
    const bf16x8 sb0 = to_bf16x8(&ds[0]), sb1 = to_bf16x8(&ds[8]);
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      f32x16 acc = zero_f32x16();
      acc = mfma32(slot_cols<D>(k_t, 0, db, lane), sb0, acc);
      acc = mfma32(slot_cols<D>(k_t, 1, db, lane), sb1, acc);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        res[0][db][j] = bf16x4{(__bf16)(acc[4 * j] * a.scale), (__bf16)(acc[4 * j + 1] * a.scale),
                               (__bf16)(acc[4 * j + 2] * a.scale), (__bf16)(acc[4 * j + 3] * a.scale)};
    }
  } else {
    // lane = key l32; register r = query acc_row(r, hi)
    f32x16 sacc = zero_f32x16(), pacc = zero_f32x16();
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      sacc = mfma32(slot_rows<D>(q_t, ks, lane), slot_rows<D>(k_t, ks, lane), sacc);
      pacc = mfma32(slot_rows<D>(do_t, ks, lane), slot_rows<D>(v_t, ks, lane), pacc);
    }
    const unsigned allow = (((kbits >> l32) & 1) ? group & vbits : 0u) >> (4 * hi);
    float p[16], ds[16];
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const f32x4 l2 = *(const VC_LDS f32x4*)(lse_slot + 8 * m + 4 * hi);
      const f32x4 d = *(const VC_LDS f32x4*)(nd_slot + 8 * m + 4 * hi);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 4 * m + i;
        const bool ok = (allow >> (8 * m + i)) & 1;
        p[r] = ok ? fast_exp2(fmaf(sacc[r], a.scale_log2, -l2[i])) : 0.0f;
        ds[r] = p[r] * (pacc[r] + d[i]);
      }
    }
    const bf16x8 pb0 = to_bf16x8(&p[0]), pb1 = to_bf16x8(&p[8]);
    const bf16x8 sb0 = to_bf16x8(&ds[0]), sb1 = to_bf16x8(&ds[8]);
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      f32x16 vacc = zero_f32x16(), kacc = zero_f32x16();
      vacc = mfma32(slot_cols<D>(do_t, 0, db, lane), pb0, vacc);
      kacc = mfma32(slot_cols<D>(q_t, 0, db, lane), sb0, kacc);
      vacc = mfma32(slot_cols<D>(do_t, 1, db, lane), pb1, vacc);
      kacc = mfma32(slot_cols<D>(q_t, 1, db, lane), sb1, kacc);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        res[0][db][j] = bf16x4{(__bf16)vacc[4 * j], (__bf16)vacc[4 * j + 1], (__bf16)vacc[4 * j + 2],
                               (__bf16)vacc[4 * j + 3]};
        res[1][db][j] = bf16x4{(__bf16)(kacc[4 * j] * a.scale), (__bf16)(kacc[4 * j + 1] * a.scale),
                               (__bf16)(kacc[4 * j + 2] * a.scale), (__bf16)(kacc[4 * j + 3] * a.scale)};
      }
    }
  }
  __syncthreads();  // every tile read of both waves is done: the tiles take the results

  // Results as rows (slot l32's row, dims db*32 + 8j + 4hi .. +3), then whole-row stores of
  // the valid slots: wave 0 dQ through the K tile, wave 1 dV through the V tile and dK
  // through the Q tile.
  auto put = [&](VC_LDS char* t, __bf16* out, const bf16x4 (&r)[D / 32][4]) {
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        *(VC_LDS bf16x4*)(t + perm_row(l32) * Tile::RS + (db * 32 + 8 * j + 4 * hi) * 2) = r[db][j];
#pragma unroll
    for (int i = 0; i < kSlots / RPI; ++i) {
      const int sl = RPI * i + lane / LPR;
      const int n = __shfl(tk, sl);
      const bf16x8 row = *(const VC_LDS bf16x8*)(t + perm_row(sl) * Tile::RS + ch * 16);
      if ((vbits >> sl) & 1) *(bf16x8*)(out + (size_t)n * tok + ch * 8) = row;
    }
  };
  if (w == 0) {
    put(k_t, a.o + base, res[0]);
  } else {
    put(v_t, a.dv + base, res[0]);
    put(q_t, a.dk + base, res[1]);
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
  const dim3 grid((unsigned)((size_t)a.B * nblk * a.H));
  const bool sum = a.sum_out != nullptr;
  if (head_dim == 128 && sum)
    hipLaunchKernelGGL((temporal_fwd_kernel<128, true>), grid, dim3(64), 0, s, a);
  else if (head_dim == 128)
    hipLaunchKernelGGL((temporal_fwd_kernel<128, false>), grid, dim3(64), 0, s, a);
  else if (sum)
    hipLaunchKernelGGL((temporal_fwd_kernel<64, true>), grid, dim3(64), 0, s, a);
  else
    hipLaunchKernelGGL((temporal_fwd_kernel<64, false>), grid, dim3(64), 0, s, a);
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
  const dim3 grid((unsigned)((size_t)a.B * nblk * a.H));
  if (head_dim == 128)
    hipLaunchKernelGGL(temporal_bwd_kernel<128>, grid, dim3(128), 0, s, a);
  else
    hipLaunchKernelGGL(temporal_bwd_kernel<64>, grid, dim3(128), 0, s, a);
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
