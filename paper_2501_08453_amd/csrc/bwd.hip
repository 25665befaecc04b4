// Backward joint text-video attention for gfx950.
//
// Prepare: per query row, -D_i = -<dO_i, O_i> and LSE_i*log2(e) in fp32, padded
//   to whole tiles of 64 rows (padding rows get LSE = +inf so that their
//   probabilities vanish, and D = 0). D is stored negated so that dP - D is
//   what the dP accumulator holds when it starts from -D.
// dK/dV (key-stationary): one workgroup of eight waves owns 256 keys of one
//   (sample, head), each wave 32, with K and V of its keys in registers and
//   dK^T, dV^T accumulated in registers. It walks over all query tiles of 64,
//   whose row-major Q and dO tiles, LSE and D are copied asynchronously
//   global -> LDS into a two-stage ring one tile ahead; one barrier per tile. Per
//   tile it recomputes S = Q K^T and P = exp2(S c log2(e) - LSE log2(e)), forms
//   dP - D = -D + dO V^T and dS = P o (dP - D) with the matrix cores, and
//   accumulates dV^T += dO^T P and dK^T += Q^T dS straight from the accumulator
//   layout (lane column = key). The transposed operands Q^T, dO^T come either
//   from transposed token tiles made by a reformatting pass (separate dQ pass)
//   or, with dQ fused in, from the row-major tiles through transposing LDS reads.
// dQ, fused (the default for joint attention at head_dim 128): in the workgroups
//   of the first key blocks (a fraction set by the host), after the dK/dV products
//   of a tile, the waves exchange dS^T through LDS (the first 32 queries in a
//   region of its own, the others over the tile's Q|dO region, dead by then) and
//   each wave computes one 32x32 block of the tile's dQ / scale = dS K over the
//   workgroup's 256 keys, with K^T held in LDS for the workgroup's lifetime. The
//   block is added to an fp32 accumulator with atomics one tile later (so that
//   the wait for the next tile's copies does not also wait for them), and the
//   workgroups of each XCD start their walk at a different query tile so that
//   concurrent atomics spread over the accumulator. For those keys S and dP are
//   computed once per (query, key) pair; the atomic traffic (fp32 dQ rows per key
//   block, performed at the memory side) is what limits the fraction: the dQ pass
//   below then covers only the other key blocks' tiles and adds the accumulator.
//   The order of the atomic additions, and so the rounding of dQ, varies from run
//   to run.
// dQ, separate (deterministic): one workgroup of eight waves owns 256 queries,
//   each wave 32, with Q^T and dO^T of its queries in registers and the lane's
//   LSE and -D as scalars. It walks over the key tiles like the forward,
//   computing S^T = K Q^T and dP^T = V dO^T, dS^T, and dQ^T += K^T dS^T with
//   dS^T taken straight from the accumulator layout (lane column = query).
//   This recomputes S and dP once more instead of scattering dQ partial sums
//   with atomics; the result is bitwise reproducible.
#include <algorithm>
#include <type_traits>

#include "common.hpp"

namespace vcja {
namespace {

constexpr int kDkdvWaves = 8;
constexpr int kBKV = 32 * kDkdvWaves;  // keys per dK/dV workgroup
static_assert(kBKV == kDkdvKeys, "dK/dV key block");
constexpr int kBQ = kTileTok;  // queries per dK/dV tile
constexpr int kDqWaves = 8;
constexpr int kDqBM = 32 * kDqWaves;  // queries per dQ workgroup
constexpr int kBN = kTileTok;         // keys per dQ tile

template <int D>
__global__ __launch_bounds__(256) void bwd_prepare_kernel(const __bf16* __restrict__ o,
                                                          const float* __restrict__ lse,
                                                          const __bf16* __restrict__ dout,
                                                          float* __restrict__ dd, float* __restrict__ lse2, int B,
                                                          int H, int N, int Npad) {
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
  }
#pragma unroll
  for (int off = 1; off < CPR; off <<= 1) sum += __shfl_xor(sum, off, 64);
  if (row < rows && chunk == 0) {
    const int h = (int)(row % H);
    const size_t bn = row / H;
    const int n = (int)(bn % N);
    const int b = (int)(bn / N);
    const size_t bh = (size_t)b * H + h;
    const float x = lse[bh * N + n];
    dd[bh * Npad + n] = -sum;
    lse2[bh * Npad + n] = (x == -INFINITY) ? INFINITY : x * kLog2e;
  }
  // Padding rows [N, Npad) of every (sample, head).
  const size_t pads = (size_t)B * H * (Npad - N);
  if (gid < pads) {
    const size_t bh = gid / (Npad - N);
    const int n = N + (int)(gid % (Npad - N));
    dd[bh * Npad + n] = 0.0f;
    lse2[bh * Npad + n] = INFINITY;
  }
}

// LDS layout of the dK/dV kernel. A stage holds one query tile: Q | dO (row-major) |
// Q^T | dO^T (transposed tiles; not with dQ fused) | LSE*log2e[64] | -D[64]. With dQ
// fused, K^T of the workgroup's keys ([D][256 + 8] bf16) follows the two stages, then
// dS^T of the tile's first 32 queries ([256 keys][32] bf16); dS^T of the other 32 is
// written over the current stage's Q | dO region once every wave is done with it.
// dS^T rows are 72 bytes (32 queries + 4 pad), and key 32u + 4j + e sits in row
// 32u + 8e + j: the writes (32 consecutive keys, one per lane) hit 64 distinct banks, the
// transposing reads (4 consecutive keys x 32 queries per half-wave) too, as the 4 keys'
// rows lie 8 apart; every address is a per-lane base plus an immediate offset.
template <int D, bool FUSED>
struct DkdvLds {
  static constexpr int RT = RowTile<D>::kBytes;
  static constexpr int TT = FUSED ? 0 : (int)tile_elems(D) * 2;
  static constexpr int STAGE = 2 * RT + 2 * TT + 512;
  static constexpr int KTS = (kBKV + 8) * 2;  // K^T row stride (bytes)
  static constexpr int DSS = (32 + 4) * 2;    // dS^T row stride (bytes)
  static constexpr int DSB = kBKV * DSS;      // dS^T of 32 queries
  static_assert(DSB <= 2 * RT, "dS^T must fit in a stage's Q | dO region");
  static constexpr int KT_OFF = 2 * STAGE;
  static constexpr int DS_OFF = KT_OFF + D * KTS;  // dS^T of the first 32 queries
  static constexpr int BYTES = FUSED ? DS_OFF + DSB : 2 * STAGE;
  // Byte offset of the 8-byte unit u (queries 4u .. 4u+3) of dS^T row j; row of key k.
  static __device__ __forceinline__ int ds_at(int j, int u) { return j * DSS + 8 * u; }
  static __device__ __forceinline__ int ds_row(int k) { return (k & ~31) | ((k & 3) << 3) | ((k >> 2) & 7); }
};

template <int D, bool SPATIAL, bool FUSED>
__global__ __launch_bounds__(64 * kDkdvWaves, 1) void bwd_dkdv_kernel(DkdvArgs a) {
  using Lds = DkdvLds<D, FUSED>;
  constexpr int RT = Lds::RT;                 // row-major Q or dO tile bytes
  constexpr int RS = RowTile<D>::kStride;     // their row stride
  constexpr int TT = Lds::TT;                 // transposed tile bytes
  constexpr int STAGE = Lds::STAGE;
  constexpr int RCOPIES = RowTile<D>::kCopies;
  constexpr int TCOPIES = TT / 1024;
  __shared__ __attribute__((aligned(1024))) char smem[Lds::BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index (uniform)
  const int l32 = lane & 31;
  const int hi = lane >> 5;
  // Spatial branch: 3-D grid (key block slot, head, sample), renumbered by XCD. Joint: 1-D
  // grid of items with the split tail dispatched last.
  int gx, h, b;
  TailItem ti{0, 0, 0, -1, 0};
  if (SPATIAL) {
    const int3 gp = xcd_grid_pos(true);
    gx = gp.x;
    h = gp.y;
    b = gp.z;
  } else {
    ti = tail_item(blockIdx.x, (a.N + kBKV - 1) / kBKV, a.H, a.B, a.tail_blocks);
    gx = ti.blk;
    h = ti.h;
    b = ti.b;
  }
  const bool tail = !SPATIAL && ti.chunk >= 0;
  const int N = a.N;
  const size_t tok = (size_t)a.H * D;
  const size_t base = (size_t)b * N * tok + (size_t)h * D;
  const size_t bh = (size_t)b * a.H + h;
  const int npad = a.ntile * kBQ;
  // Spatial branch with split text blocks: workgroups [0, text_blocks*text_chunks) of a head
  // take (text block, chunk of its query tiles) and come first in dispatch order, the rest
  // the other key blocks in order.
  int kb = gx, chunk = 0;
  bool split = false;
  if (SPATIAL && a.text_chunks > 1) {
    const int nsplit = a.text_blocks * a.text_chunks;
    split = gx < nsplit;
    kb = split ? gx % a.text_blocks : gx - nsplit + a.text_blocks;
    chunk = split ? gx / a.text_blocks : 0;
  }
  // This workgroup's keys (spatial branch: text keys, or keys of one frame).
  const RowBlock rb = row_block(kb, N, a.T, SPATIAL ? a.frame_len : 0, kBKV, true);
  const bool do_dq = FUSED && kb < a.dq_blocks;  // this key block carries its share of dQ
  const int key = rb.r0 + w * 32 + l32;  // this lane's key (accumulator column)
  const bool key_in = key < rb.r1;
  // Partial dK of this lane's key in its chunk (dV partials follow all dK partials); formed
  // only where it is written, so that no register holds it across the main loop.
  const size_t part_stride = (size_t)a.text_chunks * a.B * a.H * a.text_blocks * kBKV * D;
  auto part_k = [&]() {
    return a.text_part + ((((size_t)chunk * a.B + b) * a.H + h) * a.text_blocks * kBKV + key) * D;
  };
  // Joint tail: partial dK of this lane's key (dV partials follow all dK partials).
  const size_t tail_stride = (size_t)a.tail_blocks * a.tail_chunks * kBKV * D;
  auto tail_k = [&]() {
    return a.tail_part + (((size_t)ti.slot * a.tail_chunks + ti.chunk) * kBKV + (key - rb.r0)) * D;
  };

  AttendRule rule;
  rule.N = N;
  rule.T = a.T;
  rule.tl = a.text_len ? min(max(a.text_len[b], 0), a.T) : a.T;
  rule.L = SPATIAL ? a.frame_len : 0;
  rule.km = a.key_mask ? a.key_mask + (size_t)b * N : nullptr;
  const bool valid = key_in && rule.key_valid(key);

  if (!__syncthreads_or(valid)) {
    // No valid key in this workgroup: its dK, dV (or partials) are zero.
    if (tail) {
      const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
      float* pk = tail_k();
      for (int c = 0; c < D / 4; ++c) {
        *(f32x4*)(pk + 4 * c) = z;
        *(f32x4*)(pk + tail_stride + 4 * c) = z;
      }
    } else if (split) {
      const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
      float* pk = part_k();
      for (int c = 0; c < D / 4; ++c) {
        *(f32x4*)(pk + 4 * c) = z;
        *(f32x4*)(pk + part_stride + 4 * c) = z;
      }
    } else if (key_in) {
      const bf16x8 z = zero_bf16x8();
      for (int c = 0; c < D / 8; ++c) {
        *(bf16x8*)(a.dk + base + (size_t)key * tok + 8 * c) = z;
        *(bf16x8*)(a.dv + base + (size_t)key * tok + 8 * c) = z;
      }
    }
    return;
  }

  // Copies query tile qt into stage st. Row-major rows past N repeat row N-1; the padded
  // LSE (+inf) makes their probabilities zero.
  auto issue = [&](int qt, int st) {
    VC_LDS char* sq = (VC_LDS char*)smem + st * STAGE;
    // Spatial branch at head_dim 128: the lane index made opaque, so that the per-lane parts
    // of the copy addresses are formed here instead of held across the walk; at 256
    // registers they would be spilled, and the reload's wait, at the head of this loop,
    // would make every copy wait for the previous one.
    int cl = lane;
    if constexpr (SPATIAL && D == 128) asm volatile("" : "+v"(cl));
    for (int idx = w; idx < RCOPIES; idx += kDkdvWaves) {
      copy_row_tile<D, true, FUSED>(a.q + base, tok, qt * kBQ, N, sq, idx, cl);  // fused: perm_row order
      copy_row_tile<D, true, FUSED>(a.dout + base, tok, qt * kBQ, N, sq + RT, idx, cl);
    }
    if constexpr (!FUSED) {
      const size_t toff = (bh * a.ntile + qt) * tile_elems(D);
      for (int idx = w; idx < TCOPIES; idx += kDkdvWaves) {
        copy16_to_lds_opaque(a.qt + toff + idx * 512 + cl * 8, sq + 2 * RT + idx * 1024);
        copy16_to_lds_opaque(a.dot + toff + idx * 512 + cl * 8, sq + 2 * RT + TT + idx * 1024);
      }
    }
    // LSE*log2e by lanes 0-15, -D by lanes 16-31 of the last wave. Spatial branch: two
    // copies from uniform bases, so that no per-lane pointer is held across the walk.
    if constexpr (SPATIAL) {
      if (w == kDkdvWaves - 1) {
        const size_t r0 = bh * npad + qt * kBQ;
        if (cl < 16)
          copy16_to_lds_opaque(a.lse2 + r0 + 4 * cl, sq + 2 * RT + 2 * TT);
        else if (cl < 32)
          copy16_to_lds_opaque(a.dd + r0 + 4 * (cl - 16), sq + 2 * RT + 2 * TT);
      }
    } else if (w == kDkdvWaves - 1 && lane < 32) {
      const float* src = (lane < 16 ? a.lse2 : a.dd) + bh * npad + qt * kBQ + 4 * (lane & 15);
      copy16_to_lds_opaque(src, sq + 2 * RT + 2 * TT);
    }
  };

  // K, V of this lane's key as B operands (dims 16*ks + 8*hi .. +7).
  bf16x8 kf[D / 16], vf[D / 16];
  {
    const size_t kr = base + (size_t)min(key, rb.r1 - 1) * tok + 8 * hi;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      kf[ks] = *(const bf16x8*)(a.k + kr + 16 * ks);
      vf[ks] = *(const bf16x8*)(a.v + kr + 16 * ks);
    }
  }

  // Fused dQ: K^T of the workgroup's keys (row d holds K[key][d] of its 256 keys).
  if (FUSED && do_dq) {
    VC_LDS __bf16* ktl = (VC_LDS __bf16*)(smem + Lds::KT_OFF);
    const int kl = w * 32 + l32;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks)
#pragma unroll
      for (int t = 0; t < 8; ++t) ktl[(16 * ks + 8 * hi + t) * (Lds::KTS / 2) + kl] = kf[ks][t];
  }

  f32x16 dk_acc[D / 32], dv_acc[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) {
    dk_acc[i] = zero_f32x16();
    dv_acc[i] = zero_f32x16();
  }

  // Query tiles this workgroup visits (the same sequence for every wave): all of them in
  // joint attention; in the spatial branch the video tiles its keys are attended from.
  TileRuns runs = rule.query_tiles(rb.r0, rb.r1, a.ntile);
  if (split) {  // this chunk's part of the video query tiles
    const int c0 = a.T / kBQ + chunk * a.text_span;
    runs.b0 = max(runs.b0, c0);
    runs.b1 = min(runs.b1, c0 + a.text_span);
    if (runs.b0 >= runs.b1) runs.b1 = 0;
  }
  if (tail) {  // this chunk's run of query tiles
    runs.b0 = ti.chunk * a.tail_span;
    runs.b1 = min(a.ntile, runs.b0 + a.tail_span);
    if (runs.b0 >= runs.b1) runs.b1 = 0;
  }
  auto next_q = [&](int qt) { return (SPATIAL || tail) ? runs.next(qt) : qt; };
  // Spatial branch: a tile needs the per-pair test unless this wave's keys are all text
  // and the tile holds video queries only, or they all lie in one frame containing it.
  // (a wave past the end of a short block takes its last row)
  const int kw0 = min(rb.r0 + w * 32, rb.r1 - 1), kw1 = min(rb.r0 + w * 32 + 31, rb.r1 - 1);
  const bool wave_text_keys = kw1 < a.T;
  const int wks = SPATIAL ? rule.frame_start(kw0) : 0;
  const bool wave_one_frame = SPATIAL && kw0 >= a.T && kw1 < N && rule.frame_start(kw1) == wks;
  const int2 kr = key_range(rule, key);  // spatial: queries attending to this lane's key

  // Fused dQ: the workgroups of each XCD (dispatch is round-robin over the XCDs) start
  // their walk over the query tiles at a different eighth of them, so that the atomics
  // of concurrent workgroups land on different rows of the accumulator. Walk position u
  // visits tile phys(u).
  const int xs = (FUSED && !SPATIAL && !tail) ? (int)((blockIdx.x % kXcds) * ((a.ntile + kXcds - 1) / kXcds)) % a.ntile : 0;
  auto phys = [&](int u) { return u + xs >= a.ntile ? u + xs - a.ntile : u + xs; };
  // Fused dQ: wave w < DQ_BLOCKS forms the 32x32 block (query block dq_qb, dim block dq_db)
  // of the tile's dQ over the workgroup's 256 keys. With fewer blocks than waves (head_dim
  // 64: four), waves 0..3 take them, one per SIMD (wave w shares its SIMD with wave w + 4),
  // so that each element still gets one atomic addition per key block.
  constexpr int DQ_BLOCKS = 2 * (D / 32);
  constexpr int DQ_STEPS = kBKV / 16;
  static_assert(DQ_BLOCKS == kDkdvWaves || DQ_BLOCKS == kDkdvWaves / 2, "dQ blocks per wave");
  const bool dq_wave = DQ_BLOCKS == kDkdvWaves || w < DQ_BLOCKS;  // constant for head_dim 128
  const int dq_qb = w & 1, dq_db = (w >> 1) % (D / 32);
  f32x16 dq_blk;
  int dq_row0 = -1;  // first query row of the block awaiting its atomics, -1: none
  // The lane index as a value the compiler must treat as new at each use: per-lane
  // addresses of the fused steps derived from it are formed where they are used instead
  // of being kept in registers across the whole loop (registers are the limit here).
  auto fresh_lane = [&]() {
    int x = lane;
    asm volatile("" : "+v"(x));
    return x;
  };
  // Adds the pending dQ block to the accumulator (rows past N are padding): a uniform base
  // plus a 32-bit per-lane offset (the host launches the fused pass only when a sample's
  // N*H*D elements fit in 32 bits).
  float* const dq_dst = FUSED ? a.dq_acc + (size_t)b * N * tok + (size_t)h * D + dq_db * 32 : nullptr;
  auto flush_dq = [&]() {
    if (dq_row0 < 0) return;
    const int ln = fresh_lane();
    const int col = ln & 31, half = ln >> 5;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int qrow = dq_row0 + acc_row(r, half);
      if (qrow < N) atomicAdd(dq_dst + ((unsigned)qrow * (unsigned)tok + (unsigned)col), dq_blk[r]);
    }
    dq_row0 = -1;
  };
  // Transposing reads of the A operands Q^T, dO^T from the row-major tiles (fused: rows in
  // perm_row order): lane l of 16-lane group G supplies query 4*hi + (l%16)/4, i.e. row
  // 4*((l%16)/4) + hi, and column 16*(G%2) + 4*(l%4), relative to the operand's first query
  // row and dim block; the operand's other four queries (+8) lie 2 rows further.
  const int tr_base = (4 * ((lane & 15) >> 2) + hi) * RS + (16 * ((lane >> 4) & 1) + 4 * (lane & 3)) * 2;
  // Row of this lane's query in the plain operand reads (fused: perm_row order).
  const int prow = FUSED ? perm_row(l32) : l32;
  VC_LDS char* ds_own = (VC_LDS char*)smem + Lds::DS_OFF;

  // The walk over the query tiles; DQ: this workgroup also adds its dQ share (a separate
  // instance of the loop, so that neither carries the other's registers).
  auto walk = [&](auto dq_tag) {
    constexpr bool DQ = FUSED && decltype(dq_tag)::value;
    int qt = next_q(0);
    if (qt < a.ntile) issue(phys(qt), 0);
    for (int st = 0; qt < a.ntile; st ^= 1) {  // stage st holds tile qt, stage st ^ 1 the next
      const int qn = next_q(qt + 1);
      wait_all_memory();
      __syncthreads();  // stage st holds tile qt; every wave is done with the other stage
      if constexpr (DQ) {
        flush_dq();     // the previous tile's dQ block; waited for at the next tile
        sched_fence();  // its registers are free before the copies and products begin
      }
      if (qn < a.ntile) issue(phys(qn), st ^ 1);
      const int q0 = phys(qt) * kBQ;
      const bool pair_mask = SPATIAL && !((wave_text_keys && q0 >= a.T) ||
                                          (wave_one_frame && q0 >= wks && q0 + kBQ <= wks + rule.L));
      VC_LDS char* stage = (VC_LDS char*)smem + st * STAGE;
      const VC_LDS char* q_lds = stage;
      const VC_LDS char* do_lds = q_lds + RT;
      const VC_LDS char* qt_lds = q_lds + 2 * RT;
      const VC_LDS char* dot_lds = qt_lds + TT;
      const VC_LDS float* lse_lds = (const VC_LDS float*)(qt_lds + 2 * TT);
      const VC_LDS float* dd_lds = lse_lds + kBQ;
      bf16x8 ds_keep[2];  // fused: dS of the second query block as bf16 operands, for dQ

      auto query_block = [&](int qb) {
        f32x16 s = zero_f32x16(), dp;
  #pragma unroll
        for (int j = 0; j < 4; ++j) {  // dP accumulates on top of -D of its query rows
          const f32x4 nd = *(const VC_LDS f32x4*)(dd_lds + qb * 32 + 8 * j + 4 * hi);
  #pragma unroll
          for (int i = 0; i < 4; ++i) dp[4 * j + i] = nd[i];
        }
  #pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) {
          const bf16x8 qa = *(const VC_LDS bf16x8*)(q_lds + (qb * 32 + prow) * RS + (2 * ks + hi) * 16);
          s = mfma32(qa, kf[ks], s);
        }
  #pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) {
          const bf16x8 da = *(const VC_LDS bf16x8*)(do_lds + (qb * 32 + prow) * RS + (2 * ks + hi) * 16);
          dp = mfma32(da, vf[ks], dp);
        }
        // Register r holds query row qb*32 + 8*(r/4) + 4*hi + r%4: four runs of 4 rows.
        // Spatial branch: on tiles needing the per-pair test, queries outside [kr.x, kr.y)
        // (this lane's key range) get probability zero.
        const int row0 = pair_mask ? q0 + qb * 32 : kr.x;
        float p[16], ds[16];
  #pragma unroll
        for (int j = 0; j < 4; ++j) {
          const f32x4 l2 = *(const VC_LDS f32x4*)(lse_lds + qb * 32 + 8 * j + 4 * hi);
  #pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int r = 4 * j + i;
            p[r] = fast_exp2(fmaf(s[r], a.scale_log2, -l2[i]));
            if (SPATIAL) {
              const int qrow = row0 + acc_row(r, hi);
              p[r] = (valid & (!pair_mask | ((qrow >= kr.x) & (qrow < kr.y)))) ? p[r] : 0.0f;
            }
            // Joint attention needs no test for dK, dV: the probabilities of an invalid key
            // reach only its own lane's dK, dV, which are written as zero at the end. Its dS
            // also reaches dQ, so with dQ fused it is zeroed (its P may even be inf).
            ds[r] = p[r] * dp[r];
            if (DQ) ds[r] = valid ? ds[r] : 0.0f;
          }
        }
        // Operand element t of k-step st2 is query 16*st2 + 8*(t/4) + 4*hi + t%4: stored by
        // the transposed tiles as 8 consecutive elements at position 16*st2 + 8*hi, or read
        // from the row-major tiles by two transposing reads (rows +0..3 and +8..11).
        // Operands of the 2 * D/32 products in order (k-step st2 major, dim block db minor),
        // each read one product ahead: the read is in flight while the previous pair runs.
        constexpr int NB = D / 32;
        const int obase = (l32 * kTileRow + qb * 32 + 8 * hi) * 2;
        auto opnd = [&](int idx, const VC_LDS char* bp) {
          if constexpr (FUSED) {
            const VC_LDS char* p0 = bp + tr_base + (qb * 32 + 16 * (idx / NB)) * RS + (idx % NB) * 64;
            return cat4(lds_read_tr(p0), lds_read_tr(p0 + 2 * RS));
          } else {
            return *(const VC_LDS bf16x8*)(bp + obase + ((idx % NB) * 32 * kTileRow + 16 * (idx / NB)) * 2);
          }
        };
        if constexpr (DQ) {
          // dS^T of this query block: element t of operand st2 is query 16*st2 + 8*(t/4) +
          // 4*hi + t%4, i.e. units 4*st2 + hi and 4*st2 + 2 + hi. Block 0 goes to its own
          // region now; block 1 waits until the stage's Q and dO are no longer read.
          if (qb == 0) {
            const int ln = fresh_lane();
            const int kl = Lds::ds_row(w * 32 + (ln & 31)), hl = ln >> 5;  // dS^T row, lane half
  #pragma unroll
            for (int st2 = 0; st2 < 2; ++st2) {
              const bf16x8 x = to_bf16x8(&ds[8 * st2]);
              *(VC_LDS bf16x4*)(ds_own + Lds::ds_at(kl, 4 * st2 + hl)) = bf16x4{x[0], x[1], x[2], x[3]};
              *(VC_LDS bf16x4*)(ds_own + Lds::ds_at(kl, 4 * st2 + 2 + hl)) = bf16x4{x[4], x[5], x[6], x[7]};
            }
          }
        }
        const VC_LDS char* v_src = FUSED ? do_lds : dot_lds;
        const VC_LDS char* k_src = FUSED ? q_lds : qt_lds;
        bf16x8 av = opnd(0, v_src), ak = opnd(0, k_src);
  #pragma unroll
        for (int st2 = 0; st2 < 2; ++st2) {
          const bf16x8 pb = to_bf16x8(&p[8 * st2]);
          const bf16x8 sb = to_bf16x8(&ds[8 * st2]);
          if constexpr (DQ) ds_keep[st2] = sb;
  #pragma unroll
          for (int db = 0; db < NB; ++db) {
            const int nx = st2 * NB + db + 1;
            bf16x8 vn = av, kn = ak;
            if (nx < 2 * NB) {
              vn = opnd(nx, v_src);
              kn = opnd(nx, k_src);
            }
            dv_acc[db] = mfma32(av, pb, dv_acc[db]);
            dk_acc[db] = mfma32(ak, sb, dk_acc[db]);
            av = vn;
            ak = kn;
          }
        }
      };
  #pragma unroll 1
      for (int qb = 0; qb < kBQ / 32; ++qb) query_block(qb);

      if constexpr (DQ) {
        __syncthreads();  // every wave is done reading this stage's Q and dO
        const int ln = fresh_lane();
        {
          const int kl = Lds::ds_row(w * 32 + (ln & 31)), hl = ln >> 5;
  #pragma unroll
          for (int st2 = 0; st2 < 2; ++st2) {
            const bf16x8 x = ds_keep[st2];
            *(VC_LDS bf16x4*)(stage + Lds::ds_at(kl, 4 * st2 + hl)) = bf16x4{x[0], x[1], x[2], x[3]};
            *(VC_LDS bf16x4*)(stage + Lds::ds_at(kl, 4 * st2 + 2 + hl)) = bf16x4{x[4], x[5], x[6], x[7]};
          }
        }
        __syncthreads();  // dS^T of both query blocks complete
        if (dq_wave) {
          // dQ block: A = dS (queries x keys) by transposing reads of dS^T (this wave's query
          // block's region), B = K from K^T. Lane l of 16-lane group G supplies key
          // 16*st + 8*hi + (l%16)/4 (+4), i.e. row 32*(st/2) + 4*(st%2) + 8*((l%16)/4) + 2*hi
          // (+1), and unit 4*(G%2) + l%4 of that row.
          const VC_LDS char* ds_src = dq_qb ? (const VC_LDS char*)stage : (const VC_LDS char*)ds_own;
          const int arow = 8 * ((ln & 15) >> 2) + 2 * (ln >> 5), aunit = 4 * ((ln >> 4) & 1) + (ln & 3);
          const VC_LDS char* b_base =
              (const VC_LDS char*)smem + Lds::KT_OFF + (dq_db * 32 + (ln & 31)) * Lds::KTS + 8 * (ln >> 5) * 2;
          dq_blk = zero_f32x16();
  #pragma unroll
          for (int st = 0; st < DQ_STEPS; ++st) {
            const int j = arow + 32 * (st >> 1) + 4 * (st & 1);
            const bf16x8 da = cat4(lds_read_tr(ds_src + Lds::ds_at(j, aunit)), lds_read_tr(ds_src + Lds::ds_at(j + 1, aunit)));
            const bf16x8 kb8 = *(const VC_LDS bf16x8*)(b_base + st * 32);
            dq_blk = mfma32(da, kb8, dq_blk);
          }
          dq_row0 = q0 + dq_qb * 32;
        }
      }
      qt = qn;
    }
    if constexpr (DQ) flush_dq();
  };
  if (do_dq)
    walk(std::true_type{});
  else
    walk(std::false_type{});

  if (tail) {
    // An invalid key's partials are zero (its accumulators may hold anything).
    float* pk = tail_k();
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        f32x4 tk, tv;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          tk[e] = valid ? dk_acc[db][4 * j + e] * a.scale : 0.0f;
          tv[e] = valid ? dv_acc[db][4 * j + e] : 0.0f;
        }
        *(f32x4*)(pk + db * 32 + 8 * j + 4 * hi) = tk;
        *(f32x4*)(pk + tail_stride + db * 32 + 8 * j + 4 * hi) = tv;
      }
  } else if (split) {
    float* pk = part_k();
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4 tk = {dk_acc[db][4 * j + 0] * a.scale, dk_acc[db][4 * j + 1] * a.scale,
                          dk_acc[db][4 * j + 2] * a.scale, dk_acc[db][4 * j + 3] * a.scale};
        const f32x4 tv = {dv_acc[db][4 * j + 0], dv_acc[db][4 * j + 1], dv_acc[db][4 * j + 2], dv_acc[db][4 * j + 3]};
        *(f32x4*)(pk + db * 32 + 8 * j + 4 * hi) = tk;
        *(f32x4*)(pk + part_stride + db * 32 + 8 * j + 4 * hi) = tv;
      }
  } else if (key_in) {
    __bf16* dkp = a.dk + base + (size_t)key * tok;
    __bf16* dvp = a.dv + base + (size_t)key * tok;
    // An invalid key gets exactly zero (its accumulators may hold anything, even inf).
    auto kv = [&](float x) { return (__bf16)(valid ? x * a.scale : 0.0f); };
    auto vv = [&](float x) { return (__bf16)(valid ? x : 0.0f); };
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        bf16x4 tk = {kv(dk_acc[db][4 * j + 0]), kv(dk_acc[db][4 * j + 1]), kv(dk_acc[db][4 * j + 2]),
                     kv(dk_acc[db][4 * j + 3])};
        bf16x4 tv = {vv(dv_acc[db][4 * j + 0]), vv(dv_acc[db][4 * j + 1]), vv(dv_acc[db][4 * j + 2]),
                     vv(dv_acc[db][4 * j + 3])};
        *(bf16x4*)(dkp + db * 32 + 8 * j + 4 * hi) = tk;
        *(bf16x4*)(dvp + db * 32 + 8 * j + 4 * hi) = tv;
      }
  }
}

// Spatial branch: dK, dV of the text rows [0, nrow) as the sum of the chunks' fp32
// partials (rows = text_blocks * 256 per partial). One thread per 4 dims of one row.
template <int D>
__global__ void text_reduce_kernel(const float* part, __bf16* dk, __bf16* dv, int B, int H, int N, int rows,
                                   int nrow, int chunks) {
  const size_t total = (size_t)B * H * nrow * (D / 4);
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int d = (int)(i % (D / 4)) * 4;
  size_t t = i / (D / 4);
  const int row = (int)(t % nrow);
  t /= nrow;
  const int h = (int)(t % H);
  const int b = (int)(t / H);
  const size_t stride = (size_t)B * H * rows * D;  // one chunk
  const size_t off = (((size_t)b * H + h) * rows + row) * D + d;
  f32x4 sk = {0.0f, 0.0f, 0.0f, 0.0f}, sv = sk;
  for (int c = 0; c < chunks; ++c) {
    sk += *(const f32x4*)(part + c * stride + off);
    sv += *(const f32x4*)(part + (size_t)chunks * stride + c * stride + off);
  }
  const size_t o = (((size_t)b * N + row) * H + h) * D + d;
  *(bf16x4*)(dk + o) = bf16x4{(__bf16)sk[0], (__bf16)sk[1], (__bf16)sk[2], (__bf16)sk[3]};
  *(bf16x4*)(dv + o) = bf16x4{(__bf16)sv[0], (__bf16)sv[1], (__bf16)sv[2], (__bf16)sv[3]};
}

// Joint tail of the dK/dV kernel: dK, dV of the split items as the sum of their chunks'
// fp32 partials. One thread per 4 dims of one key row.
template <int D>
__global__ void tail_reduce_kernel(const float* part, __bf16* dk, __bf16* dv, int B, int H, int N, int items,
                                   int chunks) {
  const int nblk = (N + kBKV - 1) / kBKV;
  const size_t total = (size_t)items * kBKV * (D / 4);
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int d = (int)(i % (D / 4)) * 4;
  const int k = (int)((i / (D / 4)) % kBKV);
  const int slot = (int)(i / ((size_t)(D / 4) * kBKV));
  const int item = nblk * H * B - items + slot;
  const int row = (item % nblk) * kBKV + k;
  if (row >= N) return;
  const int h = (item / nblk) % H, b = item / (nblk * H);
  const size_t stride = (size_t)items * chunks * kBKV * D;  // dK partials, then dV
  f32x4 sk = {0.0f, 0.0f, 0.0f, 0.0f}, sv = sk;
  for (int c = 0; c < chunks; ++c) {
    const size_t off = (((size_t)slot * chunks + c) * kBKV + k) * D + d;
    sk += *(const f32x4*)(part + off);
    sv += *(const f32x4*)(part + stride + off);
  }
  const size_t o = (((size_t)b * N + row) * H + h) * D + d;
  *(bf16x4*)(dk + o) = bf16x4{(__bf16)sk[0], (__bf16)sk[1], (__bf16)sk[2], (__bf16)sk[3]};
  *(bf16x4*)(dv + o) = bf16x4{(__bf16)sv[0], (__bf16)sv[1], (__bf16)sv[2], (__bf16)sv[3]};
}

// KM: a key mask is given (a separate instance, so that the unmasked one carries none of
// its per-tile work).
template <int D, bool KM>
__global__ __launch_bounds__(64 * kDqWaves, 1) void bwd_dq_kernel(DqArgs a) {
  constexpr int RT = RowTile<D>::kBytes;      // row-major K or V tile bytes
  constexpr int RS = RowTile<D>::kStride;
  constexpr int TT = (int)tile_elems(D) * 2;  // transposed K tile bytes
  constexpr int STAGE = 2 * RT + TT;          // K | V | K^T
  constexpr int RCOPIES = RowTile<D>::kCopies;
  constexpr int TCOPIES = TT / 1024;
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index (uniform)
  const int l32 = lane & 31;
  const int hi = lane >> 5;
  // Spatial branch: 3-D grid renumbered by XCD. Joint: 1-D grid of items, split tail last.
  int gx, h, b;
  TailItem ti{0, 0, 0, -1, 0};
  if (a.frame_len) {
    const int3 gp = xcd_grid_pos(true);
    gx = gp.x;
    h = gp.y;
    b = gp.z;
  } else {
    ti = tail_item(blockIdx.x, (a.N + kDqBM - 1) / kDqBM, a.H, a.B, a.tail_blocks);
    gx = ti.blk;
    h = ti.h;
    b = ti.b;
  }
  const bool tail = ti.chunk >= 0;
  const int N = a.N;
  const size_t tok = (size_t)a.H * D;
  const size_t base = (size_t)b * N * tok + (size_t)h * D;
  const size_t bh = (size_t)b * a.H + h;
  // This workgroup's queries (spatial branch: inside one frame; text rows of dQ are written
  // by the caller's text-rows pass).
  const RowBlock rb = row_block(gx, N, a.T, a.frame_len, kDqBM, false);
  const int qi = rb.r0 + w * 32 + l32;  // this lane's query (accumulator column)
  const int qr = min(qi, rb.r1 - 1);

  // Q^T and dO^T as B operands (dims 16*ks + 8*hi .. +7), LSE*log2e and -D as scalars.
  bf16x8 qf[D / 16], dof[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    qf[ks] = *(const bf16x8*)(a.q + base + (size_t)qr * tok + 16 * ks + 8 * hi);
    dof[ks] = *(const bf16x8*)(a.dout + base + (size_t)qr * tok + 16 * ks + 8 * hi);
  }
  const float lse2 = a.lse2[bh * (size_t)a.ntile * kBN + qr];
  const float dd = a.dd[bh * (size_t)a.ntile * kBN + qr];

  f32x16 dq_acc[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) dq_acc[i] = zero_f32x16();

  AttendRule rule;
  rule.N = N;
  rule.T = a.T;
  rule.tl = a.text_len ? min(max(a.text_len[b], 0), a.T) : a.T;
  rule.L = a.frame_len;
  rule.km = a.key_mask ? a.key_mask + (size_t)b * N : nullptr;  // non-null exactly when KM
  // This wave's queries (past the end of a short block: its last row).
  const int qw0 = min(rb.r0 + w * 32, rb.r1 - 1), qw1 = min(rb.r0 + w * 32 + 31, rb.r1 - 1);
  const bool wave_all_video = qw0 >= a.T && qw1 < N;
  const int wqs = a.frame_len ? rule.frame_start(qw0) : 0;
  const bool wave_one_frame = wave_all_video && a.frame_len && rule.frame_start(qw1) == wqs;
  const QueryRange qrange = query_range(rule, qi);
  // Key tiles this workgroup visits (the same sequence for every wave).
  TileRuns runs = rule.key_tiles(rb.r0, rb.r1, a.ntile);
  const int kt0 = tail ? ti.chunk * a.tail_span : 0;  // joint tail: this chunk's key tiles
  if (tail) {
    runs.a1 = min(runs.a1, kt0 + a.tail_span);
    runs.b1 = min(runs.b1, kt0 + a.tail_span);
  }
  auto next_tile = [&](int kt) { return runs.next(kt); };
  auto issue = [&](int kt, int st) {
    VC_LDS char* sk = (VC_LDS char*)smem + st * STAGE;
    for (int idx = w; idx < RCOPIES; idx += kDqWaves) {
      copy_row_tile<D, true>(a.k + base, tok, kt * kBN, N, sk, idx, lane);
      copy_row_tile<D, true>(a.v + base, tok, kt * kBN, N, sk + RT, idx, lane);
    }
    const __bf16* tsrc = a.kt + (bh * a.ntile + kt) * tile_elems(D);
    for (int idx = w; idx < TCOPIES; idx += kDqWaves) copy16_to_lds_opaque(tsrc + idx * 512 + lane * 8, sk + 2 * RT + idx * 1024);
  };
  // The j-th copies of this wave (no-ops past the tile), issued between the score
  // products of the step's first key block: issued all at the top of the step, eight
  // waves' copies would hold up the start of every wave's matrix-core work.
  static_assert((RCOPIES + kDqWaves - 1) / kDqWaves <= D / 32 && (TCOPIES + kDqWaves - 1) / kDqWaves <= D / 32,
                "every copy of a wave needs a slot among the score products");
  auto issue_j = [&](int j, int kt, int st) {
    VC_LDS char* sk = (VC_LDS char*)smem + st * STAGE;
    const int idx = w + j * kDqWaves;
    if (idx < RCOPIES) {
      copy_row_tile<D, true>(a.k + base, tok, kt * kBN, N, sk, idx, lane);
      copy_row_tile<D, true>(a.v + base, tok, kt * kBN, N, sk + RT, idx, lane);
    }
    if (idx < TCOPIES)
      copy16_to_lds_opaque(a.kt + (bh * a.ntile + kt) * tile_elems(D) + idx * 512 + lane * 8, sk + 2 * RT + idx * 1024);
  };

  int kt = next_tile(max(kt0, a.kt_min));  // completing a fused backward: keys >= kt_min only
  if (kt < a.ntile) issue(kt, 0);
  // Key-mask bytes of each tile loaded a step ahead (waited for at the barrier with the
  // tile's copies), turned into the tile's bits there.
  int kmb = KM && kt < a.ntile ? rule.key_mask_byte(kt, lane) : 1;
  int st = 0;
  while (kt < a.ntile) {
    const int kn = next_tile(kt + 1);
    wait_all_memory();
    __syncthreads();
    const unsigned long long kbits = KM ? key_mask_bits(kmb) : ~0ull;
    if (KM && kn < a.ntile) kmb = rule.key_mask_byte(kn, lane);
    // a joint tile whose keys are all real (no padding, no text cut): masked by its bits only
    const bool plain_tile = KM && rule.L == 0 && kt * kBN + kBN <= N && (kt * kBN >= a.T || kt * kBN + kBN <= rule.tl);
    const VC_LDS char* k_lds = (const VC_LDS char*)smem + st * STAGE;
    const VC_LDS char* v_lds = k_lds + RT;
    const VC_LDS char* kt_lds = k_lds + 2 * RT;
    const int k0 = kt * kBN;
    bool need_mask;
    if (rule.km || k0 + kBN > N)
      need_mask = true;
    else if (rule.L == 0)
      need_mask = rule.tl < a.T && k0 < a.T && k0 + kBN > rule.tl;
    else if (k0 + kBN <= rule.tl)
      need_mask = !wave_all_video;
    else
      need_mask = !(wave_one_frame && k0 >= wqs && k0 + kBN <= wqs + rule.L);

#pragma unroll
    for (int kb = 0; kb < kBN / 32; ++kb) {
      f32x16 s = zero_f32x16(), dp = zero_f32x16();
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) {
        const bf16x8 ka = *(const VC_LDS bf16x8*)(k_lds + (kb * 32 + l32) * RS + (2 * ks + hi) * 16);
        s = mfma32(ka, qf[ks], s);
        if (kb == 0 && (ks & 1) && kn < a.ntile) issue_j(ks >> 1, kn, st ^ 1);
      }
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) {
        const bf16x8 va = *(const VC_LDS bf16x8*)(v_lds + (kb * 32 + l32) * RS + (2 * ks + hi) * 16);
        dp = mfma32(va, dof[ks], dp);
      }
      // Register r holds key k0 + kb*32 + 8*(r/4) + 4*hi + r%4 of this lane's query.
      float ds[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) ds[r] = fast_exp2(fmaf(s[r], a.scale_log2, -lse2));
      if (need_mask && plain_tile) {  // joint tile of real keys: the key mask's bits alone
        const unsigned bits = (unsigned)(kbits >> (32 * kb)) >> (4 * hi);
#pragma unroll
        for (int r = 0; r < 16; ++r) ds[r] = ((bits >> (8 * (r >> 2) + (r & 3))) & 1u) ? ds[r] : 0.0f;
      } else if (need_mask) {  // branch-free per element; the key mask from the tile's bits
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = k0 + kb * 32 + acc_row(r, hi);
          bool ok = KM ? rule.key_valid_bits(key, k0, kbits) : rule.key_valid(key);
          if (rule.L) ok = ok & qrange.ok(key, a.T);
          ds[r] = ok ? ds[r] : 0.0f;
        }
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) ds[r] = ds[r] * (dp[r] + dd);
#pragma unroll
      for (int st2 = 0; st2 < 2; ++st2) {
        const bf16x8 sb = to_bf16x8(&ds[8 * st2]);
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          const int off = ((db * 32 + l32) * kTileRow + kb * 32 + 16 * st2 + 8 * hi) * 2;
          dq_acc[db] = mfma32(*(const VC_LDS bf16x8*)(kt_lds + off), sb, dq_acc[db]);
        }
      }
    }
    st ^= 1;
    kt = kn;
  }

  if (tail) {  // partial dQ of this lane's query row
    float* pq = a.tail_part + (((size_t)ti.slot * a.tail_chunks + ti.chunk) * kDqBM + (qi - rb.r0)) * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4 t = {dq_acc[db][4 * j + 0] * a.scale, dq_acc[db][4 * j + 1] * a.scale,
                         dq_acc[db][4 * j + 2] * a.scale, dq_acc[db][4 * j + 3] * a.scale};
        *(f32x4*)(pq + db * 32 + 8 * j + 4 * hi) = t;
      }
  } else if (qi < rb.r1) {
    __bf16* qp = a.dq + base + (size_t)qi * tok;
    const float* fp = a.dq_acc ? a.dq_acc + base + (size_t)qi * tok : nullptr;  // the fused keys' share
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        f32x4 x = {dq_acc[db][4 * j + 0], dq_acc[db][4 * j + 1], dq_acc[db][4 * j + 2], dq_acc[db][4 * j + 3]};
        if (fp) x += *(const f32x4*)(fp + db * 32 + 8 * j + 4 * hi);
        bf16x4 t = {(__bf16)(x[0] * a.scale), (__bf16)(x[1] * a.scale), (__bf16)(x[2] * a.scale),
                    (__bf16)(x[3] * a.scale)};
        *(bf16x4*)(qp + db * 32 + 8 * j + 4 * hi) = t;
      }
  }
}

// Joint tail of the dQ kernel: dQ of the split items as the sum of their chunks' partials.
template <int D>
__global__ void tail_reduce_dq_kernel(const float* part, __bf16* dq, int B, int H, int N, int items, int chunks,
                                      const float* dq_acc, float scale) {
  const int nblk = (N + kDqBM - 1) / kDqBM;
  const size_t total = (size_t)items * kDqBM * (D / 4);
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int d = (int)(i % (D / 4)) * 4;
  const int k = (int)((i / (D / 4)) % kDqBM);
  const int slot = (int)(i / ((size_t)(D / 4) * kDqBM));
  const int item = nblk * H * B - items + slot;
  const int row = (item % nblk) * kDqBM + k;
  if (row >= N) return;
  const int h = (item / nblk) % H, b = item / (nblk * H);
  f32x4 s = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int c = 0; c < chunks; ++c) s += *(const f32x4*)(part + (((size_t)slot * chunks + c) * kDqBM + k) * D + d);
  const size_t off = (((size_t)b * N + row) * H + h) * D + d;
  if (dq_acc) s += scale * *(const f32x4*)(dq_acc + off);  // the fused keys' share (unscaled)
  *(bf16x4*)(dq + off) = bf16x4{(__bf16)s[0], (__bf16)s[1], (__bf16)s[2], (__bf16)s[3]};
}

// dq = bf16(scale * acc), four elements per thread.
__global__ void dq_from_acc_kernel(const float* acc, __bf16* dq, size_t n4, float scale) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  const f32x4 x = ((const f32x4*)acc)[i];
  ((bf16x4*)dq)[i] = bf16x4{(__bf16)(x[0] * scale), (__bf16)(x[1] * scale), (__bf16)(x[2] * scale),
                            (__bf16)(x[3] * scale)};
}

// Fused dQ: zeroes the fp32 accumulator (a kernel, not a memset, so that a captured graph
// replays it like any other node). n4 = elements / 4.
__global__ void zero_f32_kernel(float* x, size_t n4) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n4) ((f32x4*)x)[i] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
}

}  // namespace

hipError_t launch_bwd_prepare(const __bf16* o, const float* lse, const __bf16* dout, float* dd, float* lse2, int B,
                              int H, int N, int Npad, int head_dim, hipStream_t s) {
  const size_t threads = std::max((size_t)B * N * H * (head_dim / 8), (size_t)B * H * (Npad - N));
  dim3 grid((unsigned)((threads + 255) / 256));
  if (head_dim == 128)
    hipLaunchKernelGGL(bwd_prepare_kernel<128>, grid, dim3(256), 0, s, o, lse, dout, dd, lse2, B, H, N, Npad);
  else
    hipLaunchKernelGGL(bwd_prepare_kernel<64>, grid, dim3(256), 0, s, o, lse, dout, dd, lse2, B, H, N, Npad);
  return hipGetLastError();
}

hipError_t launch_bwd_dkdv(const DkdvArgs& a, int head_dim, hipStream_t s) {
  const bool spatial = a.frame_len > 0;
  const bool split = spatial && a.text_chunks > 1;
  const int nblk = row_blocks(a.N, a.T, spatial ? a.frame_len : 0, kBKV, true);
  // Spatial: 3-D grid renumbered by XCD. Joint: 1-D grid of items, the split tail last.
  dim3 grid = spatial ? dim3(nblk + (split ? (a.text_chunks - 1) * a.text_blocks : 0), a.H, a.B)
                      : dim3(nblk * a.H * a.B + a.tail_blocks * (a.tail_chunks - 1));
  const bool fused = a.dq_acc != nullptr;
  const size_t dq4 = (size_t)a.B * a.N * a.H * head_dim / 4;
  const dim3 egrid((unsigned)((dq4 + 255) / 256));
  if (fused) hipLaunchKernelGGL(zero_f32_kernel, egrid, dim3(256), 0, s, a.dq_acc, dq4);
  if (head_dim == 128 && spatial && fused)
    hipLaunchKernelGGL((bwd_dkdv_kernel<128, true, true>), grid, dim3(64 * kDkdvWaves), 0, s, a);
  else if (head_dim == 128 && spatial)
    hipLaunchKernelGGL((bwd_dkdv_kernel<128, true, false>), grid, dim3(64 * kDkdvWaves), 0, s, a);
  else if (head_dim == 128 && fused)
    hipLaunchKernelGGL((bwd_dkdv_kernel<128, false, true>), grid, dim3(64 * kDkdvWaves), 0, s, a);
  else if (head_dim == 128)
    hipLaunchKernelGGL((bwd_dkdv_kernel<128, false, false>), grid, dim3(64 * kDkdvWaves), 0, s, a);
  else if (spatial && fused)
    hipLaunchKernelGGL((bwd_dkdv_kernel<64, true, true>), grid, dim3(64 * kDkdvWaves), 0, s, a);
  else if (spatial)
    hipLaunchKernelGGL((bwd_dkdv_kernel<64, true, false>), grid, dim3(64 * kDkdvWaves), 0, s, a);
  else if (fused)
    hipLaunchKernelGGL((bwd_dkdv_kernel<64, false, true>), grid, dim3(64 * kDkdvWaves), 0, s, a);
  else
    hipLaunchKernelGGL((bwd_dkdv_kernel<64, false, false>), grid, dim3(64 * kDkdvWaves), 0, s, a);
  if (!spatial && a.tail_blocks > 0) {
    const size_t threads = (size_t)a.tail_blocks * kBKV * (head_dim / 4);
    dim3 rgrid((unsigned)((threads + 255) / 256));
    if (head_dim == 128)
      hipLaunchKernelGGL(tail_reduce_kernel<128>, rgrid, dim3(256), 0, s, a.tail_part, a.dk, a.dv, a.B, a.H, a.N,
                         a.tail_blocks, a.tail_chunks);
    else
      hipLaunchKernelGGL(tail_reduce_kernel<64>, rgrid, dim3(256), 0, s, a.tail_part, a.dk, a.dv, a.B, a.H, a.N,
                         a.tail_blocks, a.tail_chunks);
  }
  if (split) {
    const int rows = a.text_blocks * kBKV;
    const int nrow = std::min(a.T, a.N);  // the text keys
    const size_t threads = (size_t)a.B * a.H * nrow * (head_dim / 4);
    dim3 rgrid((unsigned)((threads + 255) / 256));
    if (head_dim == 128)
      hipLaunchKernelGGL(text_reduce_kernel<128>, rgrid, dim3(256), 0, s, a.text_part, a.dk, a.dv, a.B, a.H, a.N,
                         rows, nrow, a.text_chunks);
    else
      hipLaunchKernelGGL(text_reduce_kernel<64>, rgrid, dim3(256), 0, s, a.text_part, a.dk, a.dv, a.B, a.H, a.N,
                         rows, nrow, a.text_chunks);
  }
  return hipGetLastError();
}

hipError_t launch_dq_from_acc(const float* acc, __bf16* dq, size_t n, float scale, hipStream_t s) {
  const size_t n4 = n / 4;
  if (n4) hipLaunchKernelGGL(dq_from_acc_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s, acc, dq, n4, scale);
  return hipGetLastError();
}

hipError_t launch_bwd_dq(const DqArgs& a, int head_dim, hipStream_t s) {
  const int nblk = row_blocks(a.N, a.T, a.frame_len, kDqBM, false);
  // Spatial: 3-D grid renumbered by XCD. Joint: 1-D grid of items, the split tail last.
  dim3 grid = a.frame_len ? dim3(nblk, a.H, a.B) : dim3(nblk * a.H * a.B + a.tail_blocks * (a.tail_chunks - 1));
  const bool km = a.key_mask != nullptr;
  if (head_dim == 128 && km)
    hipLaunchKernelGGL((bwd_dq_kernel<128, true>), grid, dim3(64 * kDqWaves), 0, s, a);
  else if (head_dim == 128)
    hipLaunchKernelGGL((bwd_dq_kernel<128, false>), grid, dim3(64 * kDqWaves), 0, s, a);
  else if (km)
    hipLaunchKernelGGL((bwd_dq_kernel<64, true>), grid, dim3(64 * kDqWaves), 0, s, a);
  else
    hipLaunchKernelGGL((bwd_dq_kernel<64, false>), grid, dim3(64 * kDqWaves), 0, s, a);
  if (!a.frame_len && a.tail_blocks > 0) {
    const size_t threads = (size_t)a.tail_blocks * kDqBM * (head_dim / 4);
    dim3 rgrid((unsigned)((threads + 255) / 256));
    if (head_dim == 128)
      hipLaunchKernelGGL(tail_reduce_dq_kernel<128>, rgrid, dim3(256), 0, s, a.tail_part, a.dq, a.B, a.H, a.N,
                         a.tail_blocks, a.tail_chunks, a.dq_acc, a.scale);
    else
      hipLaunchKernelGGL(tail_reduce_dq_kernel<64>, rgrid, dim3(256), 0, s, a.tail_part, a.dq, a.B, a.H, a.N,
                         a.tail_blocks, a.tail_chunks, a.dq_acc, a.scale);
  }
  return hipGetLastError();
}

}  // namespace vcja
