// Temporal attention branch for long clips (33 <= F <= 144 frames) on gfx950.
//
// Each spatial position l of a (sample, head) attends across its F frames, the rows
// T + f*L + l of the joint [B, N, H, D] layout (Sec. III-B regroups [B, F, L, ...] as
// [B*L, F, ...]). Sequences this long no longer fit one 32-slot matrix-core block, so a
// workgroup takes one position at a time and splits its frames into blocks of 32, each
// wave walking the other side's blocks for its own block(s), two at a time with the
// products of the pair interleaved (one block's chain of matrix-core ops alone leaves
// the loop bound by its latency).
//
// The work is bound by memory traffic (about 0.25 KiB per row and head each way against
// a few hundred flops per byte of matrix work). A persistent workgroup per compute unit
// walks a strided sequence of positions (head fastest, so that concurrent workgroups read
// whole token rows together).
//   Forward: two buffers of K | V rows; while position p is computed from one, the
//     rows of p+1 are copied into the other. Wave j owns query block j.
//   Backward: the four row tiles Q | K | V | dO of one position at once (156 KiB at 144
//     frames: no second buffer fits). D_i = <dO_i, O_i> (no preparation pass, no
//     workspace), LSE_i and the valid-key bits are formed first; waves 0-4 then form
//     dK, dV of one key block each and waves 5-7 dQ of the query blocks; the results
//     leave as whole rows through the tiles.
// Rows sit in LDS in the permuted order of the fused joint backward (frame 16g + 4m + i
// in row 16g + 4i + m) with a 16-byte pad chunk per row, so that the transposing reads of
// four consecutive frames hit distinct banks; reads past the last frame are clamped to it
// (their probabilities are zero), so a position needs F rows of LDS, not 32*ceil(F/32).
#include <algorithm>

#include "common.hpp"

namespace vcja {
namespace {

constexpr int kLongWaves = 8;
constexpr int kLongMaxBlocks = (kMaxTemporalFramesLong + 31) / 32;  // frame blocks of 32
constexpr int kLongPadRows = (kMaxTemporalFramesLong + 15) / 16 * 16;

template <int D>
struct LongLds {
  static constexpr int CH = D / 8 + 1;   // 16-byte chunks per row, pad included
  static constexpr int RS = CH * 16;     // row stride (bytes)
  // 1 KiB wave copies of one tensor's rows (kLongPadRows rows), and its LDS region
  static constexpr int COPIES = (kLongPadRows * CH + 63) / 64;
  static constexpr int REGION = COPIES * 1024;
  static constexpr int STATS = 2 * 32 * kLongMaxBlocks * 4;  // LSE*log2e | -D per query slot
  static constexpr int BYTES = 4 * REGION + STATS;
};

// The lane index as a value the compiler must treat as new where it is taken: per-lane
// addresses derived from it are then formed in each phase instead of being hoisted out of
// the position loop and kept (or spilled) across it.
__device__ __forceinline__ int opaque_lane() {
  int x = threadIdx.x & 63;
  asm volatile("" : "+v"(x));
  return x;
}

// The rows (frames) of one position of one tensor: frame f at src + f * fstride.
struct PosRows {
  const __bf16* src;
  size_t fstride;
};

// Issues this wave's share of the copies of rows [0, round_up(F, 16)) into `dst` in
// permuted order (LDS row r holds frame perm_row(r), clamped to the last frame).
template <int D, int NW = kLongWaves>
__device__ __forceinline__ void copy_rows(PosRows pr, int F, VC_LDS char* dst, int w) {
  constexpr int CH = LongLds<D>::CH;
  const int lane = opaque_lane();
  const int rows = (F + 15) & ~15;
  const int copies = (rows * CH + 63) / 64;
  for (int idx = w; idx < copies; idx += NW) {
    const int lin = idx * 64 + lane;
    const int r = lin / CH;
    const int c = min(lin - r * CH, CH - 2);
    const int f = min(perm_row(r), F - 1);
    copy16_to_lds_opaque(pr.src + (size_t)f * pr.fstride + c * 8, dst + idx * 1024);
  }
}

// Byte offset in a region of the 16-byte chunk `chunk` of frame t (clamped to F-1).
template <int D>
__device__ __forceinline__ int row_off(int t, int F) {
  return perm_row(min(t, F - 1)) * LongLds<D>::RS;
}

// A operand of a product whose contraction runs over frames (X^T, m = dim, k = frame):
// dims db*32 + l32, frames 16*st + 8*(t/4) + 4*hi + t%4 (t = 0..7) of block `blk`, the
// order an accumulator column holds them; two transposing reads of 4 frames each. Each
// lane supplies the address of frame r0 + e (e = (lane%16)/4, clamped) and 4 dims.
template <int D>
__device__ __forceinline__ bf16x8 frames_operand(const VC_LDS char* region, int blk, int st, int db, int F,
                                                 int lane) {
  const int hi = lane >> 5;
  const int e = (lane & 15) >> 2;
  const int col = (db * 32 + 16 * ((lane >> 4) & 1) + 4 * (lane & 3)) * 2;
  const int r0 = blk * 32 + 16 * st + 4 * hi + e;
  const bf16x4 a = lds_read_tr(region + row_off<D>(r0, F) + col);
  const bf16x4 b = lds_read_tr(region + row_off<D>(r0 + 8, F) + col);
  return cat4(a, b);
}

// A operand of a product whose contraction runs over dims (X rows, m = frame, k = dim):
// frame blk*32 + l32, dims 16*ks + 8*hi .. +7.
template <int D>
__device__ __forceinline__ bf16x8 rows_operand(const VC_LDS char* region, int blk, int ks, int F, int lane) {
  const int l32 = lane & 31, hi = lane >> 5;
  return *(const VC_LDS bf16x8*)(region + row_off<D>(blk * 32 + l32, F) + (2 * ks + hi) * 16);
}

// Position item i: head fastest, then spatial position, then sample.
struct PosItem {
  int b, l, h;
};
__device__ __forceinline__ PosItem pos_item(int i, int H, int L) { return PosItem{i / (H * L), (i / H) % L, i % H}; }

// Key validity of the 32 frames of block `blk` of the position starting at `kbase`
// (frame f at kbase + f*L of the sample's key_mask row), as a bit mask (wave-uniform).
__device__ __forceinline__ unsigned key_bits(const uint8_t* km, int kbase, int L, int F, int blk, int lane) {
  const int f = blk * 32 + (lane & 31);
  bool ok = f < F;
  if (km) ok = ok & (km[kbase + (size_t)min(f, F - 1) * L] != 0);
  return (unsigned)__ballot(ok);
}

template <int D, bool SUM>
__global__ __launch_bounds__(64 * kLongWaves, 1) void temporal_long_fwd_kernel(TemporalArgs a) {
  using Lds = LongLds<D>;
  __shared__ __attribute__((aligned(1024))) char smem[Lds::BYTES];
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int F = a.F, L = a.L, H = a.H;
  const int nblk = (F + 31) / 32;
  const size_t tok = (size_t)H * D;
  const int items = a.B * L * H;
  auto rows_of = [&](const __bf16* t, PosItem it) {
    return PosRows{t + ((size_t)it.b * a.N + a.T + it.l) * tok + (size_t)it.h * D, (size_t)L * tok};
  };
  auto issue = [&](int i, int buf) {
    const PosItem it = pos_item(i, H, L);
    VC_LDS char* dst = (VC_LDS char*)smem + buf * 2 * Lds::REGION;
    copy_rows<D>(rows_of(a.k, it), F, dst, w);
    copy_rows<D>(rows_of(a.v, it), F, dst + Lds::REGION, w);
  };

  // This wave's query rows (B operands: the lane's frame w*32 + l32, clamped to the last
  // frame, dims 16*ks + 8*hi..), loaded one item ahead so that their latency overlaps the
  // previous item's work.
  auto load_q = [&](int i, bf16x8* dst) {
    const PosItem it = pos_item(i, H, L);
    const int ln = opaque_lane();
    const size_t row = ((size_t)it.b * a.N + a.T + (size_t)min(w * 32 + (ln & 31), F - 1) * L + it.l) * tok +
                       (size_t)it.h * D + 8 * (ln >> 5);
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) dst[ks] = *(const bf16x8*)(a.q + row + 16 * ks);
  };
  bf16x8 qf[D / 16], qn[D / 16];
  int buf = 0;
  if ((int)blockIdx.x < items) {
    issue(blockIdx.x, 0);
    if (w < nblk) load_q(blockIdx.x, qf);
  }
  for (int i = blockIdx.x; i < items; i += gridDim.x, buf ^= 1) {
    wait_all_memory();
    __syncthreads();  // K, V of item i are in buffer `buf`; nobody reads the other buffer
    const bool more = i + (int)gridDim.x < items;
    if (more) issue(i + gridDim.x, buf ^ 1);
    if (w >= nblk) continue;  // no query block for this wave
    if (more) load_q(i + gridDim.x, qn);
    const PosItem it = pos_item(i, H, L);
    const int lane = opaque_lane();
    const int l32 = lane & 31, hi = lane >> 5;
    const VC_LDS char* kr = (const VC_LDS char*)smem + buf * 2 * Lds::REGION;
    const VC_LDS char* vr = kr + Lds::REGION;
    const uint8_t* km = a.key_mask ? a.key_mask + (size_t)it.b * a.N + a.T + it.l : nullptr;
    // This lane's query: frame q of the wave's block (past F: the last frame, not written).
    const int q = w * 32 + l32;
    const bool q_in = q < F;
    f32x16 oacc[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db) oacc[db] = zero_f32x16();
    float m = -INFINITY, l = 0.0f;  // base (log2 units) and this half's sum
    // Key blocks two at a time (the score products of both interleaved, one rescale of the
    // running base for the pair), then the odd one.
    auto scores = [&](int kb, unsigned bits, f32x16& s, float& mx) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[r] = ((bits >> acc_row(r, hi)) & 1u) ? s[r] * a.scale_log2 : -INFINITY;
        mx = fmaxf(mx, s[r]);
      }
    };
    auto rebase = [&](float mx) {
      const float m_new = fmaxf(m, halves_max(mx));
      const float alpha = fast_exp2(m - m_new);  // m = -inf at the first block: 0
      m = m_new;
      l *= alpha;
#pragma unroll
      for (int db = 0; db < D / 32; ++db) oacc[db] *= alpha;
    };
    auto pv = [&](int kb, const f32x16& s) {
      float p[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        p[r] = fast_exp2(s[r] - m);
        l += p[r];
      }
      const bf16x8 pb0 = to_bf16x8(&p[0]), pb1 = to_bf16x8(&p[8]);
#pragma unroll
      for (int db = 0; db < D / 32; ++db) {
        oacc[db] = mfma32(frames_operand<D>(vr, kb, 0, db, F, lane), pb0, oacc[db]);
        oacc[db] = mfma32(frames_operand<D>(vr, kb, 1, db, F, lane), pb1, oacc[db]);
      }
    };
    int kb = 0;
    for (; kb + 1 < nblk; kb += 2) {
      const unsigned bits0 = key_bits(km, 0, L, F, kb, lane), bits1 = key_bits(km, 0, L, F, kb + 1, lane);
      if ((bits0 | bits1) == 0) continue;  // no valid key in either block (uniform)
      f32x16 s0 = zero_f32x16(), s1 = zero_f32x16();
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) {
        s0 = mfma32(rows_operand<D>(kr, kb, ks, F, lane), qf[ks], s0);
        s1 = mfma32(rows_operand<D>(kr, kb + 1, ks, F, lane), qf[ks], s1);
      }
      float mx = -INFINITY;
      scores(kb, bits0, s0, mx);
      scores(kb + 1, bits1, s1, mx);
      rebase(mx);
      pv(kb, s0);
      pv(kb + 1, s1);
    }
    if (kb < nblk) {
      const unsigned bits = key_bits(km, 0, L, F, kb, lane);
      if (bits != 0) {
        f32x16 s = zero_f32x16();
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) s = mfma32(rows_operand<D>(kr, kb, ks, F, lane), qf[ks], s);
        float mx = -INFINITY;
        scores(kb, bits, s, mx);
        rebase(mx);
        pv(kb, s);
      }
    }
    const float lt = halves_sum(l);
    const float inv = lt > 0.0f ? 1.0f / lt : 0.0f;
    if (q_in) {
      const size_t orow = ((size_t)it.b * a.N + a.T + (size_t)q * L + it.l) * tok + (size_t)it.h * D;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int d = db * 32 + 8 * j + 4 * hi;
          const bf16x4 o4 = {(__bf16)(oacc[db][4 * j + 0] * inv), (__bf16)(oacc[db][4 * j + 1] * inv),
                             (__bf16)(oacc[db][4 * j + 2] * inv), (__bf16)(oacc[db][4 * j + 3] * inv)};
          *(bf16x4*)(a.o + orow + d) = o4;
          if constexpr (SUM) {  // out = (o_joint + o_spatial) + o in fp32, rounded once
            f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
            if (a.sum_a) {
              const bf16x4 x = *(const bf16x4*)(a.sum_a + orow + d);
#pragma unroll
              for (int e = 0; e < 4; ++e) acc[e] += (float)x[e];
            }
            if (a.sum_b) {
              const bf16x4 x = *(const bf16x4*)(a.sum_b + orow + d);
#pragma unroll
              for (int e = 0; e < 4; ++e) acc[e] += (float)x[e];
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[e] += (float)o4[e];
            *(bf16x4*)(a.sum_out + orow + d) = bf16x4{(__bf16)acc[0], (__bf16)acc[1], (__bf16)acc[2], (__bf16)acc[3]};
          }
        }
      if (hi == 0)
        a.lse[((size_t)it.b * H + it.h) * a.N + a.T + (size_t)q * L + it.l] =
            lt > 0.0f ? (m + __log2f(lt)) * kLn2 : -INFINITY;
    }
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) qf[ks] = qn[ks];
  }
}

// Result rows of frame block `blk` (lane l32's frame blk*32 + l32, dims db*32 + 8j + 4hi ..
// +3 in res[db][j]) into a tile, then whole-row stores of the block's frames < F to
// dst + f*fstride. The wave reads back only rows it wrote (LDS operations of a wave complete
// in order).
template <int D>
__device__ __forceinline__ void put_block_rows(VC_LDS char* t, __bf16* dst, size_t fstride, int blk, int F,
                                               const bf16x4 (&res)[D / 32][4]) {
  constexpr int LPR = D / 8, RPI = 64 / LPR;
  int lane = opaque_lane();
  const int f = blk * 32 + (lane & 31);
  if (f < F) {
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        *(VC_LDS bf16x4*)(t + row_off<D>(f, F) + (db * 32 + 8 * j + 4 * (lane >> 5)) * 2) = res[db][j];
  }
  lane = opaque_lane();
#pragma unroll
  for (int i = 0; i < 32 / RPI; ++i) {
    const int fr = blk * 32 + RPI * i + lane / LPR;
    if (fr < F)
      *(bf16x8*)(dst + (size_t)fr * fstride + (lane % LPR) * 8) =
          *(const VC_LDS bf16x8*)(t + row_off<D>(fr, F) + (lane % LPR) * 16);
  }
}

// Backward: one position at a time per workgroup (persistent), all four row tiles Q | K | V
// | dO of the position resident in LDS. D = <dO, O> (O read as whole rows while the tiles
// fill), LSE*log2(e) and the valid-key bits of every frame are formed first and shared
// through LDS. Wave j < 5 forms dK, dV of key block j (lane = key: S, dP from -D,
// dV^T += dO^T P, dK^T += Q^T dS over the query blocks); waves 5, 6, 7 form dQ of query
// blocks j - 5 and j - 2 (lane = query: S^T, dP^T, dS^T, dQ^T += K^T dS^T over the key
// blocks), so that each SIMD carries about the same matrix work. The results go back
// through the tiles (dQ through K, dK through Q, dV through V) so that every global store
// is a whole 16-byte chunk of a row; the next position's copies go out once every wave has
// read its rows back, so they overlap those stores. One full wait per position.
template <int D>
__global__ __launch_bounds__(64 * kLongWaves, 1) void temporal_long_bwd_kernel(TemporalArgs a) {
  using Lds = LongLds<D>;
  constexpr int NW = kLongWaves;
  constexpr int LPR = D / 8;     // lanes per row in a whole-row access
  constexpr int RPI = 64 / LPR;  // rows per whole-row wave access
  constexpr int NOI = ((kLongPadRows + RPI - 1) / RPI + NW - 1) / NW;  // O row loads per wave
  constexpr int KBW = 32 * kLongMaxBlocks / 16;  // words of valid-key bits (16 frames each)
  __shared__ __attribute__((aligned(1024))) char smem[Lds::BYTES + 4 * KBW];
  VC_LDS char* const q_t = (VC_LDS char*)smem;
  VC_LDS char* const k_t = q_t + Lds::REGION;
  VC_LDS char* const v_t = k_t + Lds::REGION;
  VC_LDS char* const do_t = v_t + Lds::REGION;
  VC_LDS float* const lse_s = (VC_LDS float*)(smem + 4 * Lds::REGION);  // LSE*log2e per frame slot
  VC_LDS float* const nd_s = lse_s + 32 * kLongMaxBlocks;               // -D per frame slot
  VC_LDS unsigned* const kbits = (VC_LDS unsigned*)(smem + Lds::BYTES);  // valid keys, 16 frames per word
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int F = a.F, L = a.L, H = a.H;
  const int nblk = (F + 31) / 32;
  const size_t tok = (size_t)H * D;
  const size_t fstride = (size_t)L * tok;  // frame stride of a position's rows
  const int items = a.B * L * H;
  const bool kv_role = w < kLongMaxBlocks;  // dK, dV of key block w; else dQ of blocks m, m + 3
  const int m = w - kLongMaxBlocks;
  auto block_bits = [&](int blk) { return kbits[2 * blk] | (kbits[2 * blk + 1] << 16); };

  for (int i = blockIdx.x; i < items; i += gridDim.x) {
    const PosItem it = pos_item(i, H, L);
    const size_t base = ((size_t)it.b * a.N + a.T + it.l) * tok + (size_t)it.h * D;  // frame 0's row
    const size_t rbase = ((size_t)it.b * H + it.h) * a.N + a.T + it.l;              // frame 0's LSE
    __syncthreads();  // every wave has read back the previous position's results
    copy_rows<D, NW>(PosRows{a.q + base, fstride}, F, q_t, w);
    copy_rows<D, NW>(PosRows{a.k + base, fstride}, F, k_t, w);
    copy_rows<D, NW>(PosRows{a.v + base, fstride}, F, v_t, w);
    copy_rows<D, NW>(PosRows{a.dout + base, fstride}, F, do_t, w);
    // O rows (whole-row loads; frames past F clamped, their D unused), and the LSE and
    // key-mask byte of frames 16w .. 16w + 15 and, past 16*NW, 16(w + NW) .. (clamped
    // likewise; the mask byte from any readable byte if there is no mask). Every load here
    // is used only after the full wait below.
    int lane = opaque_lane();
    const int ch = lane % LPR;
    bf16x8 of[NOI];
#pragma unroll
    for (int j = 0; j < NOI; ++j) {
      const int r = min((w + NW * j) * RPI + lane / LPR, F - 1);
      of[j] = *(const bf16x8*)(a.o_in + base + (size_t)r * fstride + ch * 8);
    }
    constexpr int NF = (KBW + NW - 1) / NW;  // 16-frame groups per wave
    float lse_v[NF];
    int kmb[NF];
#pragma unroll
    for (int g = 0; g < NF; ++g) {
      const int f = min(16 * (w + NW * g) + (lane & 15), F - 1);
      lse_v[g] = a.lse[rbase + (size_t)f * L];
      kmb[g] = *(a.key_mask ? a.key_mask + (size_t)it.b * a.N + a.T + it.l + (size_t)f * L : (const uint8_t*)a.lse);
    }
    wait_all_memory();
#pragma unroll
    for (int g = 0; g < NF; ++g) asm volatile("" : "+v"(kmb[g]), "+v"(lse_v[g]));  // uses stay after the wait
    __syncthreads();  // the position's rows are in LDS
    lane = opaque_lane();
    // -D per frame slot (0 past F), LSE*log2e (+inf past F or where a frame has no valid
    // key), valid-key bits
#pragma unroll
    for (int j = 0; j < NOI; ++j) {
      const int r = (w + NW * j) * RPI + lane / LPR;
      if (r < 32 * nblk) {  // whole groups of LPR lanes
        float acc = 0.0f;
        if (r < F) {
          const bf16x8 dv = *(const VC_LDS bf16x8*)(do_t + row_off<D>(r, F) + ch * 16);
#pragma unroll
          for (int e = 0; e < 8; ++e) acc = fmaf((float)dv[e], (float)of[j][e], acc);
        }
#pragma unroll
        for (int s = 1; s < LPR; s <<= 1) acc += __shfl_xor(acc, s);
        if (ch == 0) nd_s[r] = r < F ? -acc : 0.0f;
      }
    }
#pragma unroll
    for (int g = 0; g < NF; ++g) {
      const int grp = w + NW * g;
      const int f = 16 * grp + (lane & 15);
      if (grp < KBW) {
        if (lane < 16 && f < 32 * nblk) lse_s[f] = (f < F && lse_v[g] != -INFINITY) ? lse_v[g] * kLog2e : INFINITY;
        const unsigned kb = (unsigned)__ballot(f < F && (!a.key_mask || kmb[g] != 0)) & 0xffffu;
        if (lane == 0) kbits[grp] = kb;
      }
    }
    __syncthreads();  // statistics and key bits of every frame are in LDS

    const int l32 = lane & 31, hi = lane >> 5;
    bf16x4 r0[D / 32][4], r1[D / 32][4];  // key waves: dK, dV; query waves: dQ of block m in r0
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) r0[db][j] = r1[db][j] = bf16x4{};
    if (kv_role) {
      if (w < nblk) {
        // ---- lane = key w*32 + l32 ----
        const bool valid = ((block_bits(w) >> l32) & 1u) != 0;
        bf16x8 kf[D / 16], vf[D / 16];
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) {
          kf[ks] = rows_operand<D>(k_t, w, ks, F, lane);
          vf[ks] = rows_operand<D>(v_t, w, ks, F, lane);
        }
        f32x16 dk[D / 32], dv[D / 32];
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          dk[db] = zero_f32x16();
          dv[db] = zero_f32x16();
        }
        for (int qb = 0; qb < nblk; ++qb) {
          const int ln = opaque_lane();
          f32x16 s = zero_f32x16(), dp;
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {  // dP accumulates on top of -D of its query rows
            const f32x4 nd = *(const VC_LDS f32x4*)(nd_s + qb * 32 + 8 * jj + 4 * hi);
#pragma unroll
            for (int e = 0; e < 4; ++e) dp[4 * jj + e] = nd[e];
          }
#pragma unroll
          for (int ks = 0; ks < D / 16; ++ks) {
            s = mfma32(rows_operand<D>(q_t, qb, ks, F, ln), kf[ks], s);
            dp = mfma32(rows_operand<D>(do_t, qb, ks, F, ln), vf[ks], dp);
          }
          // An invalid key's P and dS reach only its own lane's dK, dV, written as zero.
          bf16x8 pb[2], sb[2];
#pragma unroll
          for (int h2 = 0; h2 < 2; ++h2) {
            float p[8], ds[8];
#pragma unroll
            for (int jj = 0; jj < 2; ++jj) {
              const f32x4 l2 = *(const VC_LDS f32x4*)(lse_s + qb * 32 + 8 * (2 * h2 + jj) + 4 * hi);
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const int r = 8 * h2 + 4 * jj + e;
                p[4 * jj + e] = fast_exp2(fmaf(s[r], a.scale_log2, -l2[e]));
                ds[4 * jj + e] = p[4 * jj + e] * dp[r];
              }
            }
            pb[h2] = to_bf16x8(p);
            sb[h2] = to_bf16x8(ds);
          }
          sched_fence();
#pragma unroll
          for (int db = 0; db < D / 32; ++db) {
            dv[db] = mfma32(frames_operand<D>(do_t, qb, 0, db, F, ln), pb[0], dv[db]);
            dv[db] = mfma32(frames_operand<D>(do_t, qb, 1, db, F, ln), pb[1], dv[db]);
          }
          sched_fence();
#pragma unroll
          for (int db = 0; db < D / 32; ++db) {
            dk[db] = mfma32(frames_operand<D>(q_t, qb, 0, db, F, ln), sb[0], dk[db]);
            dk[db] = mfma32(frames_operand<D>(q_t, qb, 1, db, F, ln), sb[1], dk[db]);
          }
        }
        const float ks_ = valid ? a.scale : 0.0f, vs_ = valid ? 1.0f : 0.0f;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            r0[db][jj] = bf16x4{(__bf16)(dk[db][4 * jj] * ks_), (__bf16)(dk[db][4 * jj + 1] * ks_),
                                (__bf16)(dk[db][4 * jj + 2] * ks_), (__bf16)(dk[db][4 * jj + 3] * ks_)};
            r1[db][jj] = bf16x4{(__bf16)(dv[db][4 * jj] * vs_), (__bf16)(dv[db][4 * jj + 1] * vs_),
                                (__bf16)(dv[db][4 * jj + 2] * vs_), (__bf16)(dv[db][4 * jj + 3] * vs_)};
          }
      }
    } else {
      // ---- lane = query qb*32 + l32, qb = m and m + 3 ----
      auto dq_block = [&](int qb, f32x16 (&dq)[D / 32]) {
        const int q = qb * 32 + l32;
        bf16x8 qf[D / 16], dof[D / 16];
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) {
          qf[ks] = rows_operand<D>(q_t, qb, ks, F, lane);
          dof[ks] = rows_operand<D>(do_t, qb, ks, F, lane);
        }
        const float l2 = lse_s[q];
        const float nd = nd_s[q];
#pragma unroll
        for (int db = 0; db < D / 32; ++db) dq[db] = zero_f32x16();
        // Key blocks two at a time (their products interleaved, so that each chain of
        // matrix-core ops has the other's to overlap), then the odd one.
        auto sdp = [&](int kb, f32x16& s, f32x16& dp, int ln, int ks) {
          s = mfma32(rows_operand<D>(k_t, kb, ks, F, ln), qf[ks], s);
          dp = mfma32(rows_operand<D>(v_t, kb, ks, F, ln), dof[ks], dp);
        };
        auto grad = [&](int kb, const f32x16& s, const f32x16& dp, bf16x8& sb0, bf16x8& sb1) {
          const unsigned bits = block_bits(kb);
          float ds[16];
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float p = ((bits >> acc_row(r, hi)) & 1u) ? fast_exp2(fmaf(s[r], a.scale_log2, -l2)) : 0.0f;
            ds[r] = p * (dp[r] + nd);
          }
          sb0 = to_bf16x8(&ds[0]);
          sb1 = to_bf16x8(&ds[8]);
        };
        auto acc = [&](int kb, bf16x8 sb0, bf16x8 sb1, int ln) {
#pragma unroll
          for (int db = 0; db < D / 32; ++db) {
            dq[db] = mfma32(frames_operand<D>(k_t, kb, 0, db, F, ln), sb0, dq[db]);
            dq[db] = mfma32(frames_operand<D>(k_t, kb, 1, db, F, ln), sb1, dq[db]);
          }
        };
        int kb = 0;
        for (; kb + 1 < nblk; kb += 2) {
          const int ln = opaque_lane();
          f32x16 s0 = zero_f32x16(), dp0 = zero_f32x16(), s1 = zero_f32x16(), dp1 = zero_f32x16();
#pragma unroll
          for (int ks = 0; ks < D / 16; ++ks) {
            sdp(kb, s0, dp0, ln, ks);
            sdp(kb + 1, s1, dp1, ln, ks);
          }
          bf16x8 a0, a1, b0, b1;
          grad(kb, s0, dp0, a0, a1);
          grad(kb + 1, s1, dp1, b0, b1);
          acc(kb, a0, a1, ln);
          acc(kb + 1, b0, b1, ln);
        }
        if (kb < nblk) {
          const int ln = opaque_lane();
          f32x16 s0 = zero_f32x16(), dp0 = zero_f32x16();
#pragma unroll
          for (int ks = 0; ks < D / 16; ++ks) sdp(kb, s0, dp0, ln, ks);
          bf16x8 a0, a1;
          grad(kb, s0, dp0, a0, a1);
          acc(kb, a0, a1, ln);
        }
      };
      // Block m + 3 first, stored straight from the accumulator (8-byte pieces), so that
      // only block m's results are held across the barrier below.
      if (m + 3 < nblk) {
        f32x16 dq[D / 32];
        dq_block(m + 3, dq);
        const int q = (m + 3) * 32 + l32;
        if (q < F) {
#pragma unroll
          for (int db = 0; db < D / 32; ++db)
#pragma unroll
            for (int j = 0; j < 4; ++j)
              *(bf16x4*)(a.o + base + (size_t)q * fstride + db * 32 + 8 * j + 4 * hi) =
                  bf16x4{(__bf16)(dq[db][4 * j] * a.scale), (__bf16)(dq[db][4 * j + 1] * a.scale),
                         (__bf16)(dq[db][4 * j + 2] * a.scale), (__bf16)(dq[db][4 * j + 3] * a.scale)};
        }
      }
      if (m < nblk) {
        f32x16 dq[D / 32];
        dq_block(m, dq);
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            r0[db][j] = bf16x4{(__bf16)(dq[db][4 * j] * a.scale), (__bf16)(dq[db][4 * j + 1] * a.scale),
                               (__bf16)(dq[db][4 * j + 2] * a.scale), (__bf16)(dq[db][4 * j + 3] * a.scale)};
      }
    }
    __syncthreads();  // every wave is done reading the tiles: they take the results

    if (kv_role) {
      if (w < nblk) {
        put_block_rows<D>(q_t, a.dk + base, fstride, w, F, r0);
        put_block_rows<D>(v_t, a.dv + base, fstride, w, F, r1);
      }
    } else if (m < nblk) {
      put_block_rows<D>(k_t, a.o + base, fstride, m, F, r0);
    }
  }
  wait_all_memory();  // no copy or load of this workgroup outlives it
}

}  // namespace

hipError_t launch_temporal_long_fwd(const TemporalArgs& a, int head_dim, int cus, hipStream_t s) {
  const int items = a.B * a.L * a.H;
  dim3 grid((unsigned)std::max(1, std::min(items, cus)));
  const bool sum = a.sum_out != nullptr;
  if (head_dim == 128 && sum)
    hipLaunchKernelGGL((temporal_long_fwd_kernel<128, true>), grid, dim3(64 * kLongWaves), 0, s, a);
  else if (head_dim == 128)
    hipLaunchKernelGGL((temporal_long_fwd_kernel<128, false>), grid, dim3(64 * kLongWaves), 0, s, a);
  else if (sum)
    hipLaunchKernelGGL((temporal_long_fwd_kernel<64, true>), grid, dim3(64 * kLongWaves), 0, s, a);
  else
    hipLaunchKernelGGL((temporal_long_fwd_kernel<64, false>), grid, dim3(64 * kLongWaves), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_temporal_long_bwd(const TemporalArgs& a, int head_dim, int cus, hipStream_t s) {
  const int items = a.B * a.L * a.H;
  dim3 grid((unsigned)std::max(1, std::min(items, cus)));
  if (head_dim == 128)
    hipLaunchKernelGGL(temporal_long_bwd_kernel<128>, grid, dim3(64 * kLongWaves), 0, s, a);
  else
    hipLaunchKernelGGL(temporal_long_bwd_kernel<64>, grid, dim3(64 * kLongWaves), 0, s, a);
  return hipGetLastError();
}

}  // namespace vcja
