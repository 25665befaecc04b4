// Forward joint text-video attention for gfx950.
//
// One workgroup of eight waves owns 256 queries of one (sample, head); each
// wave owns 32 of them, held in registers. Keys stream through LDS as
// row-major tiles of 64 (rows padded by 16 bytes) and values as transposed
// token tiles (prepared by a reformatting pass), both copied asynchronously
// global -> LDS. Scores read the K tile one step before the P V products read
// the V^T tile of the same keys, so each has its own two-slot ring (tile t in
// slot t mod 2): the copies of step j+1 are in flight during step j, and one
// barrier per tile suffices. All eight waves share each tile. Each wave issues its
// share of those copies between its score products rather than all at the top of
// the step, where eight waves' worth of copy instructions would stall the start of
// the matrix-core work.
//
// The wave computes the transposed score block S^T = K Q^T with 32x32x16 bf16
// matrix-core steps, so each lane's accumulator column is one query: the
// running maximum and sum of the online softmax are per-lane scalars that need
// one exchange between the two wave halves per tile. P^T leaves the
// accumulator already laid out as the B operand of O^T += V^T P^T, so
// probabilities never go through LDS.
//
// Software pipeline inside each wave: at step j the matrix cores get the
// scores of tile j+1 and then O += P_j V_j back to back, and the softmax of
// tile j+1 runs on the vector ALUs while the P_j V_j products execute.
//
// The online softmax keeps a per-query exponent base m and does not take the
// tile maximum on the common path: probabilities are formed against the
// current base and summed (in the bf16 precision the P V product uses, two at
// a time); only when a lane's sum of 32 probabilities exceeds 2^13 (or is not
// finite, e.g. before the first valid key) does the wave raise the base to the
// tile maximum and recompute the tile. Probabilities therefore stay below
// 2^13 and the O rescale, which must wait for the products in flight, is rare.
// The log-sum-exp is kept for the recomputing backward.
#include "common.hpp"

namespace vcja {
namespace {

constexpr int kWaves = 8;
constexpr int kWavesPerSimd = 2;  // register budget: two waves share each SIMD
constexpr int kBM = 32 * kWaves;  // queries per workgroup
constexpr int kBN = kTileTok;     // keys per tile
constexpr float kSumLimit = 8192.0f;  // largest accepted sum of a lane's 32 probabilities

template <int D>
struct FwdTile {
  static constexpr int KT = RowTile<D>::kBytes;       // K tile bytes
  static constexpr int KS = RowTile<D>::kStride;      // K row stride
  static constexpr int VTB = (int)tile_elems(D) * 2;  // V^T tile bytes
  static constexpr int LDS = 2 * KT + 2 * VTB;        // K ring | V^T ring
};

struct NoHook {
  __device__ void operator()(int) const {}
};

// S^T (keys x queries) of one 64-key tile: two 32x32 blocks, A = K rows from LDS,
// B = this wave's Q^T fragments, K fragments read two k-steps ahead of their products.
// hook(j) runs after k-step 2j+1 (j < D/32).
template <int D, class Hook = NoHook>
__device__ __forceinline__ void scores(const VC_LDS char* ks_lds, const bf16x8* qf, int l32, int hi, f32x16* s,
                                       Hook hook = Hook()) {
  constexpr int KS = FwdTile<D>::KS;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) s[kb] = zero_f32x16();
  constexpr int KSN = D / 16;
  bf16x8 f[KSN][2];
  auto rd = [&](int ks) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) f[ks][kb] = *(const VC_LDS bf16x8*)(ks_lds + (kb * 32 + l32) * KS + (2 * ks + hi) * 16);
  };
  rd(0);
  rd(1);
#pragma unroll
  for (int ks = 0; ks < KSN; ++ks) {
    sched_fence();
    if (ks + 2 < KSN) rd(ks + 2);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) s[kb] = mfma32(f[ks][kb], qf[ks], s[kb]);
    if (ks & 1) hook(ks >> 1);
  }
  sched_fence();
}

// O^T += V^T P^T for one 64-key tile. Operand element t of k-step st2 (lane half hi) is
// key 16*st2 + 8*(t/4) + 4*hi + t%4, stored by the transposed tile as 8 consecutive
// elements at position 16*st2 + 8*hi.
template <int D>
__device__ __forceinline__ void accumulate_pv(const VC_LDS char* vt_lds, const bf16x8* pb, int l32, int hi,
                                              f32x16* oacc) {
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int st2 = 0; st2 < 2; ++st2)
#pragma unroll
      for (int db = 0; db < D / 32; ++db) {
        const bf16x8 af =
            *(const VC_LDS bf16x8*)(vt_lds + ((db * 32 + l32) * kTileRow + kb * 32 + 16 * st2 + 8 * hi) * 2);
        oacc[db] = mfma32(af, pb[2 * kb + st2], oacc[db]);
      }
}

// Masking of one wave's score tiles (lane = query qi).
struct KeyMask {
  AttendRule rule;
  QueryRange qr;        // spatial: keys this lane's query attends to
  bool wave_all_video;  // spatial: every query of the wave is a video row (< N)
  bool wave_one_frame;  // spatial: ... and they all lie in the frame starting at wqs
  int wqs;
  __device__ __forceinline__ bool tile_needs_mask(int k0) const {
    const AttendRule& r = rule;
    if (r.km || k0 + kBN > r.N) return true;
    if (r.L == 0) return r.tl < r.T && k0 < r.T && k0 + kBN > r.tl;
    if (k0 + kBN <= r.tl) return !wave_all_video;  // real text keys only
    return !(wave_one_frame && k0 >= wqs && k0 + kBN <= wqs + r.L);
  }
  // Sets scores of keys this lane's query does not attend to to -inf. Branch-free per
  // element: the tests are plain arithmetic, the key mask the tile's bits
  // (key_mask_bits).
  template <bool KM>
  __device__ __forceinline__ void apply(f32x16* s, int k0, int hi, unsigned long long kbits) const {
    if (KM && rule.L == 0 && k0 + kBN <= rule.N && (k0 >= rule.T || k0 + kBN <= rule.tl)) {
      // Joint tile of real keys (no padding, no text cut): the key mask's bits alone.
      // Register r of key block kb holds key kb*32 + 8*(r/4) + 4*hi + r%4 of the tile.
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const unsigned bits = (unsigned)(kbits >> (32 * kb)) >> (4 * hi);
#pragma unroll
        for (int r = 0; r < 16; ++r) s[kb][r] = ((bits >> (8 * (r >> 2) + (r & 3))) & 1u) ? s[kb][r] : -INFINITY;
      }
      return;
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = k0 + kb * 32 + acc_row(r, hi);
        bool ok = KM ? rule.key_valid_bits(key, k0, kbits) : rule.key_valid(key);
        if (rule.L) ok = ok & qr.ok(key, rule.T);
        s[kb][r] = ok ? s[kb][r] : -INFINITY;
      }
  }
};

// Sum of eight bf16 values (two at a time, fp32 accumulation) added to sum.
__device__ __forceinline__ float add_bf16x8(bf16x8 x, float sum) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
  for (int i = 0; i < 4; ++i) sum = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{x[2 * i], x[2 * i + 1]}, ones, sum, false);
  return sum;
}

// Probabilities 2^(s c log2(e) - m) of 8 scores (one PV operand), rounded to bf16, with
// their sum added to sum.
__device__ __forceinline__ bf16x8 probs8(const f32x16& s, int half, float scale_log2, float m, float& sum) {
  float p[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) p[t] = fast_exp2(fmaf(s[8 * half + t], scale_log2, -m));
  const bf16x8 r = to_bf16x8(p);
  sum = add_bf16x8(r, sum);
  return r;
}

// Rare path: raises the exponent base of the queries (lanes) that need it to the tile
// maximum (both wave halves agree), recomputes the tile's probabilities and their sum,
// and returns the factor that rescales what was accumulated against the old base.
__device__ __forceinline__ float raise_base(const f32x16* s, float scale_log2, bool need, float& m, bf16x8* pb,
                                            float& psum) {
  float mx[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) mx[c] = fmaxf(s[c >> 1][8 * (c & 1)], s[c >> 1][8 * (c & 1) + 1]);
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int t = 2; t < 8; ++t) mx[c] = fmaxf(mx[c], s[c >> 1][8 * (c & 1) + t]);
  const float tmax = halves_max(fmaxf(fmaxf(mx[0], mx[1]), fmaxf(mx[2], mx[3]))) * scale_log2;
  need = need | (swap_halves(need ? 1.0f : 0.0f) != 0.0f);
  const float m_new = need ? fmaxf(m, tmax) : m;
  const float alpha = m_new == m ? 1.0f : fast_exp2(m - m_new);
  m = m_new;
  const float m_use = m == -INFINITY ? 0.0f : m;  // no valid key yet: all probabilities 0
  psum = 0.0f;
#pragma unroll
  for (int c = 0; c < 4; ++c) pb[c] = probs8(s[c >> 1], c & 1, scale_log2, m_use, psum);
  return alpha;
}

// V^T operand fragments of PV chunk c (key block c/2, k-step c%2) for every dim block.
template <int D>
__device__ __forceinline__ void load_vt_chunk(const VC_LDS char* vt_lds, int c, int l32, int hi, bf16x8* f) {
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
    f[db] = *(const VC_LDS bf16x8*)(vt_lds + ((db * 32 + l32) * kTileRow + (c >> 1) * 32 + 16 * (c & 1) + 8 * hi) * 2);
}

// KM: a key mask is given (a separate instance, so that the unmasked one carries none of
// its per-tile work).
template <int D, bool KM>
__global__ __launch_bounds__(64 * kWaves, kWavesPerSimd * 4 / kWaves) void fwd_kernel(FwdArgs a) {
  constexpr int KT = FwdTile<D>::KT;
  constexpr int VTB = FwdTile<D>::VTB;
  constexpr int KCOPIES = RowTile<D>::kCopies;  // 1 KiB wave copies per tile
  constexpr int VCOPIES = VTB / 1024;
  static_assert(VTB % 1024 == 0, "transposed tile must be whole wave copies");
  __shared__ __attribute__((aligned(1024))) char smem[FwdTile<D>::LDS];

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
    ti = tail_item(blockIdx.x, (a.N + kBM - 1) / kBM, a.H, a.B, a.tail_blocks);
    gx = ti.blk;
    h = ti.h;
    b = ti.b;
  }
  const bool tail = ti.chunk >= 0;
  const int N = a.N;
  const size_t tok = (size_t)a.H * D;
  const size_t base = (size_t)b * N * tok + (size_t)h * D;
  const __bf16* vt_bh = a.vt + ((size_t)b * a.H + h) * a.ntile * tile_elems(D);
  // This workgroup's queries (spatial branch: inside one frame; text rows are written
  // by the caller's text-rows pass).
  const RowBlock rb = row_block(gx, N, a.T, a.frame_len, kBM, false);
  const int qi = rb.r0 + w * 32 + l32;
  const bool q_in = qi < rb.r1;

  // Q^T as the B operand: lane holds query qi, dims 16*ks + 8*hi .. +7.
  bf16x8 qf[D / 16];
  {
    const __bf16* qp = a.q + base + (size_t)min(qi, rb.r1 - 1) * tok + 8 * hi;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) qf[ks] = *(const bf16x8*)(qp + 16 * ks);
  }

  KeyMask mask;
  mask.rule.N = N;
  mask.rule.T = a.T;
  mask.rule.tl = a.text_len ? min(max(a.text_len[b], 0), a.T) : a.T;
  mask.rule.L = a.frame_len;
  mask.rule.km = a.key_mask ? a.key_mask + (size_t)b * N : nullptr;  // non-null exactly when KM
  mask.qr = query_range(mask.rule, qi);
  {
    // This wave's queries; a wave past the end of a short block takes its last row, so that
    // it follows the same tile path as the others.
    const int qw0 = min(rb.r0 + w * 32, rb.r1 - 1), qw1 = min(rb.r0 + w * 32 + 31, rb.r1 - 1);
    mask.wave_all_video = qw0 >= a.T && qw1 < N;
    mask.wqs = a.frame_len ? mask.rule.frame_start(qw0) : 0;
    mask.wave_one_frame = mask.wave_all_video && a.frame_len && mask.rule.frame_start(qw1) == mask.wqs;
  }
  // Key tiles this workgroup visits (the same sequence for every wave): all but tiles of
  // padded text only in joint attention; text and own-frame tiles in the spatial branch.
  TileRuns runs = mask.rule.key_tiles(rb.r0, rb.r1, a.ntile);
  const int kt0 = tail ? ti.chunk * a.tail_span : 0;  // joint tail: this chunk's key tiles
  if (tail) {
    runs.a1 = min(runs.a1, kt0 + a.tail_span);
    runs.b1 = min(runs.b1, kt0 + a.tail_span);
  }
  auto next_tile = [&](int kt) { return runs.next(kt); };
  // Copies tile kt's K rows (rows past N repeat row N-1 and are masked) or V^T tile into
  // ring slot `slot`. The copies are issued through inline assembly, so the compiler
  // neither waits for them nor lets them force full waits on LDS reads; the kernel waits
  // for them itself (wait_all_memory) before the barrier after which they are read.
  auto issue_k = [&](int kt, int slot) {
    VC_LDS char* dst = (VC_LDS char*)smem + slot * KT;
    for (int idx = w; idx < KCOPIES; idx += kWaves) copy_row_tile<D, true>(a.k + base, tok, kt * kBN, N, dst, idx, lane);
  };
  auto issue_v = [&](int kt, int slot) {
    VC_LDS char* dst = (VC_LDS char*)smem + 2 * KT + slot * VTB;
    const __bf16* vsrc = vt_bh + (size_t)kt * tile_elems(D);
    for (int idx = w; idx < VCOPIES; idx += kWaves) copy16_to_lds_opaque(vsrc + idx * 512 + lane * 8, dst + idx * 1024);
  };
  // The j-th K or V^T copy of this wave (a no-op past the tile), issued from the score
  // loop's hook.
  static_assert((KCOPIES + kWaves - 1) / kWaves <= D / 32 && (VCOPIES + kWaves - 1) / kWaves <= D / 32,
                "every copy of a wave needs a hook slot");
  auto k_copy = [&](int j, int kt, int slot) {
    const int idx = w + j * kWaves;
    if (idx < KCOPIES) copy_row_tile<D, true>(a.k + base, tok, kt * kBN, N, (VC_LDS char*)smem + slot * KT, idx, lane);
  };
  auto v_copy = [&](int j, int kt, int slot) {
    const int idx = w + j * kWaves;
    if (idx < VCOPIES)
      copy16_to_lds_opaque(vt_bh + (size_t)kt * tile_elems(D) + idx * 512 + lane * 8,
                           (VC_LDS char*)smem + 2 * KT + slot * VTB + idx * 1024);
  };
  auto k_slot = [&](int slot) { return (const VC_LDS char*)smem + slot * KT; };
  auto v_slot = [&](int slot) { return (const VC_LDS char*)smem + 2 * KT + slot * VTB; };

  f32x16 oacc[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) oacc[i] = zero_f32x16();
  float m = -INFINITY;  // exponent base (scaled scores, log2 units)
  float l = 0.0f;       // running sum of this lane's half
  bf16x8 pb[4];         // probabilities of the current tile as PV operands

  int cur = next_tile(kt0);
  if (cur < a.ntile) {
    int nxt = next_tile(cur + 1);
    int par = 0;  // ring slot of tile `cur`
    issue_k(cur, 0);
    issue_v(cur, 0);
    if (nxt < a.ntile) issue_k(nxt, 1);
    // Key-mask bytes of `cur` now and of each next tile a step ahead: their waits are the
    // ones before the barriers (a byte loaded and used in the same step would wait for the
    // step's tile copies too).
    const int kmb_cur = KM ? mask.rule.key_mask_byte(cur, lane) : 1;
    int kmb_nxt = KM && nxt < a.ntile ? mask.rule.key_mask_byte(nxt, lane) : 1;
    wait_all_memory();
    __syncthreads();
    // Prologue: scores and softmax of the first tile.
    {
      f32x16 s[2];
      scores<D>(k_slot(0), qf, l32, hi, s);
      if (mask.tile_needs_mask(cur * kBN)) mask.apply<KM>(s, cur * kBN, hi, KM ? key_mask_bits(kmb_cur) : ~0ull);
      raise_base(s, a.scale_log2, true, m, pb, l);
    }
    // Pending rescale of O: probabilities computed against a raised base must only be
    // added after O is brought to that base (done before the next P V, so that the
    // P V products of the current tile and the softmax of the next share one branch-free
    // stretch of code).
    float alpha = 1.0f;
    bool raise = false;
    // Steady state: scores of `nxt` and P V of `cur` on the matrix cores, softmax of
    // `nxt` on the vector ALUs.
    while (nxt < a.ntile) {
      const int nn = next_tile(nxt + 1);
      wait_all_memory();
      __syncthreads();  // K of `nxt` and V^T of `cur` landed; K of `cur` and V^T of the
                        // previous tile are no longer read by any wave
      const unsigned long long kbits = KM ? key_mask_bits(kmb_nxt) : ~0ull;  // key mask of `nxt`
      if (KM && nn < a.ntile) kmb_nxt = mask.rule.key_mask_byte(nn, lane);
      if (__any(raise)) {
#pragma unroll
        for (int i = 0; i < D / 32; ++i) oacc[i] *= alpha;
      }
      f32x16 s[2];
      // The copies of this step go to the slots freed by the barrier: K of `nn` to the
      // slot of K of `cur`, V^T of `nxt` to the slot of the previous V^T tile.
      scores<D>(k_slot(par ^ 1), qf, l32, hi, s, [&](int j) {
        if (nn < a.ntile) k_copy(j, nn, par);
        v_copy(j, nxt, par ^ 1);
      });
      if (mask.tile_needs_mask(nxt * kBN)) mask.apply<KM>(s, nxt * kBN, hi, kbits);
      // P V of `cur` in four chunks of D/32 products; between them the vector ALUs do
      // the softmax of `nxt`: first its new base, then one operand's probabilities per
      // chunk. Fragments of the next chunk are read one chunk ahead.
      const VC_LDS char* vt_lds = v_slot(par);
      bf16x8 fa[D / 32], fb[D / 32];
      load_vt_chunk<D>(vt_lds, 0, l32, hi, fa);
      float psum = 0.0f;
      bf16x8 pn[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        sched_fence();
        if (c < 3) load_vt_chunk<D>(vt_lds, c + 1, l32, hi, fb);
#pragma unroll
        for (int db = 0; db < D / 32; ++db) oacc[db] = mfma32(fa[db], pb[c], oacc[db]);
        pn[c] = probs8(s[c >> 1], c & 1, a.scale_log2, m, psum);
        if (c < 3) {  // the next chunk's reads first, then products and softmax interleaved
          __builtin_amdgcn_sched_group_barrier(0x100, D / 32, 0);
#pragma unroll
          for (int db = 0; db < D / 32; ++db) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);
          }
        }
#pragma unroll
        for (int db = 0; db < D / 32; ++db) fa[db] = fb[db];
      }
      sched_fence();
      const bool need = !(psum <= kSumLimit);
      alpha = 1.0f;
      raise = __any(need);
      if (raise) alpha = raise_base(s, a.scale_log2, need, m, pn, psum);
#pragma unroll
      for (int c = 0; c < 4; ++c) pb[c] = pn[c];
      l = fmaf(l, alpha, psum);
      par ^= 1;
      cur = nxt;
      nxt = nn;
    }
    if (__any(raise)) {
#pragma unroll
      for (int i = 0; i < D / 32; ++i) oacc[i] *= alpha;
    }
    wait_all_memory();
    __syncthreads();  // V^T of the last tile landed
    accumulate_pv<D>(v_slot(par), pb, l32, hi, oacc);
  }

  const float lt = halves_sum(l);
  const float inv = lt > 0.0f ? 1.0f / lt : 0.0f;
  if (tail) {  // this chunk's unnormalised O, base and sum for the merge
    const size_t rows = (size_t)a.tail_blocks * a.tail_chunks * kBM;
    const size_t row = ((size_t)ti.slot * a.tail_chunks + ti.chunk) * kBM + (qi - rb.r0);
    float* po = a.tail_part + row * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4 t = {oacc[db][4 * j + 0], oacc[db][4 * j + 1], oacc[db][4 * j + 2], oacc[db][4 * j + 3]};
        *(f32x4*)(po + db * 32 + 8 * j + 4 * hi) = t;
      }
    if (hi == 0) {
      a.tail_part[rows * D + row] = m;
      a.tail_part[rows * D + rows + row] = lt;
    }
  } else if (q_in) {
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

// Joint tail: O and LSE of the split items from their chunks' partials,
// O = sum_c 2^(m_c - M) O_c / sum_c 2^(m_c - M) l_c over the chunks that saw a valid key
// (M the largest of their bases). One thread per 4 dims of one query row.
template <int D>
__global__ void tail_merge_kernel(const float* part, __bf16* o, float* lse, int B, int H, int N, int items,
                                  int chunks) {
  const int nblk = (N + kBM - 1) / kBM;
  const size_t total = (size_t)items * kBM * (D / 4);
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int d = (int)(i % (D / 4)) * 4;
  const int k = (int)((i / (D / 4)) % kBM);
  const int slot = (int)(i / ((size_t)(D / 4) * kBM));
  const int item = nblk * H * B - items + slot;
  const int row = (item % nblk) * kBM + k;
  if (row >= N) return;
  const int h = (item / nblk) % H, b = item / (nblk * H);
  const size_t rows = (size_t)items * chunks * kBM;
  const float* pm = part + rows * D;
  const float* pl = pm + rows;
  float mx = -INFINITY;
  for (int c = 0; c < chunks; ++c) {
    const size_t r = ((size_t)slot * chunks + c) * kBM + k;
    if (pl[r] > 0.0f) mx = fmaxf(mx, pm[r]);
  }
  float sum = 0.0f;
  f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int c = 0; c < chunks; ++c) {
    const size_t r = ((size_t)slot * chunks + c) * kBM + k;
    if (pl[r] > 0.0f) {
      const float wgt = exp2f(pm[r] - mx);
      sum += wgt * pl[r];
      acc += wgt * *(const f32x4*)(part + r * D + d);
    }
  }
  const float inv = sum > 0.0f ? 1.0f / sum : 0.0f;
  const size_t off = (((size_t)b * N + row) * H + h) * D + d;
  *(bf16x4*)(o + off) = bf16x4{(__bf16)(acc[0] * inv), (__bf16)(acc[1] * inv), (__bf16)(acc[2] * inv),
                               (__bf16)(acc[3] * inv)};
  if (d == 0) lse[((size_t)b * H + h) * N + row] = sum > 0.0f ? (mx + log2f(sum)) * kLn2 : -INFINITY;
}

}  // namespace

hipError_t launch_fwd(const FwdArgs& a, int head_dim, hipStream_t s) {
  const int nblk = row_blocks(a.N, a.T, a.frame_len, kBM, false);
  // Spatial: 3-D grid renumbered by XCD. Joint: 1-D grid of items, the split tail last.
  dim3 grid = a.frame_len ? dim3(nblk, a.H, a.B) : dim3(nblk * a.H * a.B + a.tail_blocks * (a.tail_chunks - 1));
  const bool km = a.key_mask != nullptr;
  if (head_dim == 128 && km)
    hipLaunchKernelGGL((fwd_kernel<128, true>), grid, dim3(64 * kWaves), 0, s, a);
  else if (head_dim == 128)
    hipLaunchKernelGGL((fwd_kernel<128, false>), grid, dim3(64 * kWaves), 0, s, a);
  else if (km)
    hipLaunchKernelGGL((fwd_kernel<64, true>), grid, dim3(64 * kWaves), 0, s, a);
  else
    hipLaunchKernelGGL((fwd_kernel<64, false>), grid, dim3(64 * kWaves), 0, s, a);
  if (!a.frame_len && a.tail_blocks > 0) {
    const size_t threads = (size_t)a.tail_blocks * kBM * (head_dim / 4);
    dim3 rgrid((unsigned)((threads + 255) / 256));
    if (head_dim == 128)
      hipLaunchKernelGGL(tail_merge_kernel<128>, rgrid, dim3(256), 0, s, a.tail_part, a.o, a.lse, a.B, a.H, a.N,
                         a.tail_blocks, a.tail_chunks);
    else
      hipLaunchKernelGGL(tail_merge_kernel<64>, rgrid, dim3(256), 0, s, a.tail_part, a.o, a.lse, a.B, a.H, a.N,
                         a.tail_blocks, a.tail_chunks);
  }
  return hipGetLastError();
}

}  // namespace vcja
