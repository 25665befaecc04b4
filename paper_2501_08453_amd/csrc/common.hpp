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

constexpr int kTileTok = 64;  // tokens per tile (keys or queries) in every kernel
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

#define VC_LDS __attribute__((address_space(3)))
typedef short i16x4 __attribute__((ext_vector_type(4)));

// Asynchronous 16-byte copy global -> LDS: lane t of the wave writes its 16 bytes at
// lds_wave_base + 16*t (lds_wave_base must be the same for the whole wave). Completion is
// tracked by the vector-memory counter.
__device__ __forceinline__ void copy16_to_lds(const void* g, VC_LDS void* lds_wave_base) {
  __builtin_amdgcn_global_load_lds(g, lds_wave_base, 16, 0, 0);
}

// The same copy issued through inline assembly. The compiler then does not know that the
// instruction writes LDS, so it inserts no wait for it before later LDS reads: it would
// otherwise wait for every copy in flight before any read whose address it cannot prove
// distinct from the copies' (the ring's other stage, in practice). The caller waits for
// the copies (wait_all_memory) before reading what they write. Sets M0; a kernel using it
// must issue all of its LDS copies this way, so that nothing else relies on M0.
__device__ __forceinline__ void copy16_to_lds_opaque(const void* g, VC_LDS void* lds_wave_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :
               : "s"((unsigned)(size_t)lds_wave_base), "v"(g)
               : "memory");
}

// Waits for every outstanding memory operation of this wave (vector memory and LDS).
__device__ __forceinline__ void wait_all_memory() { __builtin_amdgcn_s_waitcnt(0); }

// Transposing LDS read (ds_read_b64_tr_b16). Within each group of 16 lanes, lane 4e+g
// supplies the address of 4 consecutive bf16 at (row r0+e, columns c0+4g .. c0+4g+3) of a
// row-major tile; lane i of the group receives the column c0+i of rows r0 .. r0+3.
__device__ __forceinline__ bf16x4 lds_read_tr(const VC_LDS void* p) {
  i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((VC_LDS i16x4*)p);
  return __builtin_bit_cast(bf16x4, v);
}

// Row-major bf16 tile of 64 token rows x D in LDS with one 16-byte pad chunk per row:
// row stride D*2 + 16 bytes, so the 16 rows read by one quarter-wave at a common column
// fall on distinct banks, and every k-step of an operand read is an immediate offset
// from one per-lane base address.
template <int D>
struct RowTile {
  static constexpr int kChunks = D / 8 + 1;             // 16-byte chunks per row, pad included
  static constexpr int kStride = kChunks * 16;          // bytes per row
  static constexpr int kBytes = kTileTok * kStride;     // bytes per tile
  static constexpr int kCopies = kTileTok * kChunks / 64;  // 1 KiB wave copies per tile
  static_assert(kTileTok * kChunks % 64 == 0, "tile must be whole wave copies");
};

// Row order of a permuted row tile: token 16g + 4m + i of the tile sits in LDS row
// 16g + 4i + m (a 4x4 transpose inside each run of 16; its own inverse). Four consecutive
// tokens then lie 4 rows apart, so that a transposing read of them (4 rows x 64 bytes per
// half-wave) hits 64 distinct banks, while 16 consecutive tokens still occupy 16 distinct
// rows of the run for the plain 16-byte reads.
__host__ __device__ constexpr int perm_row(int t) { return (t & ~15) | ((t & 3) << 2) | ((t >> 2) & 3); }

// Issues wave copy `idx` of a row tile: rows row0 .. row0+63 of the [B, N, H, D] tensor
// slice at src (row r at src + r*tok), rows clamped to N-1. The pad chunk of each row
// repeats the row's last chunk. PERM: the tile's rows in perm_row order.
template <int D, bool OPAQUE = false, bool PERM = false>
__device__ __forceinline__ void copy_row_tile(const __bf16* src, size_t tok, int row0, int N, VC_LDS char* dst,
                                              int idx, int lane) {
  constexpr int CH = RowTile<D>::kChunks;
  const int lin = idx * 64 + lane;
  const int r = lin / CH;
  const int c = min(lin - r * CH, CH - 2);
  const __bf16* g = src + (size_t)min(row0 + (PERM ? perm_row(r) : r), N - 1) * tok + c * 8;
  if constexpr (OPAQUE)
    copy16_to_lds_opaque(g, dst + idx * 1024);
  else
    copy16_to_lds(g, dst + idx * 1024);
}

// Scheduling hint for the basic block it ends: issue `lead` LDS reads, then `n` times
// {1 matrix-core op, 1 LDS read, v vector-ALU ops}, so that independent vector work
// (softmax, elementwise gradients) executes while the matrix core is busy.
template <int lead, int n, int v>
__device__ __forceinline__ void interleave_mfma_valu() {
  __builtin_amdgcn_sched_group_barrier(0x100, lead, 0);
#pragma unroll
  for (int i = 0; i < n; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, v, 0);
  }
}

// Bits of a tile's key mask from the lanes' bytes (AttendRule::key_mask_byte): bit i = the
// byte of lane i is non-zero. Wave-uniform.
__device__ __forceinline__ unsigned long long key_mask_bits(int byte) { return __ballot(byte != 0); }

// Value of lane l^32 (the other half of the wave).
__device__ __forceinline__ float swap_halves(float x) { return __shfl_xor(x, 32, 64); }

// max / sum of x over lanes l and l^32.
__device__ __forceinline__ float halves_max(float x) { return fmaxf(x, swap_halves(x)); }
__device__ __forceinline__ float halves_sum(float x) { return x + swap_halves(x); }

// Keeps the compiler from moving any instruction across this point.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

// Transposed token tiles ("token-major" copies). A [B, N, H, D] tensor X is also kept as
// blocked tiles XT[b][h][tile][d][kTileRow] of kTileTok tokens: row d of a tile holds
// X[tile*64 + tok][d] for the 64 tokens, followed by 8 padding elements (so that the 32
// rows read by one MFMA operand fall on distinct LDS banks). Inside each run of 16 tokens
// the second and third groups of 4 are swapped, so that the 8 tokens a lane supplies to
// one 32x32x16 MFMA step - tokens 16s + 8*(t/4) + 4*hi + t%4, t = 0..7, the order in
// which an accumulator column holds them - are 8 consecutive elements (one 16-byte read).
constexpr int kTileRow = kTileTok + 8;  // elements per transposed tile row
__host__ __device__ constexpr size_t tile_elems(int d) { return (size_t)d * kTileRow; }
// Position of token t (0..63) inside a transposed tile row.
__host__ __device__ constexpr int tok_pos(int t) {
  return (t & ~15) | (((t >> 2) & 3) == 1 ? 8 : ((t >> 2) & 3) == 2 ? 4 : ((t >> 2) & 3) * 4) | (t & 3);
}

// Joint attention runs a 1-D grid of items (row block, head, sample), row block fastest.
// The last `tail_items` items, those of the last, partial round of dispatch, are replaced by
// tail_chunks workgroups each, dispatched after all others, every one over a run of tiles
// along the other token axis; the round then ends after about 1/tail_chunks of the time.
struct TailItem {
  int blk, h, b;  // row block, head, sample
  int chunk;      // -1: a whole item; else the run of tiles [chunk*span, (chunk+1)*span)
  int slot;       // tail: index of the item among the split ones
};
__device__ __forceinline__ TailItem tail_item(int x, int nblk, int H, int B, int tail_items) {
  const int regular = nblk * H * B - tail_items;
  int item = x, chunk = -1, slot = 0;
  if (x >= regular) {
    slot = (x - regular) % tail_items;
    chunk = (x - regular) / tail_items;
    item = regular + slot;
  }
  return TailItem{item % nblk, (item / nblk) % H, item / (nblk * H), chunk, slot};
}

// The rows (queries or keys) a workgroup owns, [r0, r1), at most `per` of them. Joint
// attention: uniform blocks over [0, N). Spatial branch: no block straddles a frame or the
// text slot (a straddling block would visit the key tiles of two frames, each wave masking
// half of them): first the text rows [0, T) in blocks (with `text`: the key side), then
// ceil(L / per) blocks per frame, the last one shorter when `per` does not divide L.
struct RowBlock {
  int r0, r1;
};
__host__ __device__ inline int row_blocks(int N, int T, int L, int per, bool text) {
  if (L == 0) return (N + per - 1) / per;
  return (text ? (T + per - 1) / per : 0) + ((N - T) / L) * ((L + per - 1) / per);
}
__device__ __forceinline__ RowBlock row_block(int x, int N, int T, int L, int per, bool text) {
  if (L == 0) return RowBlock{x * per, min(N, (x + 1) * per)};
  const int tb = text ? (T + per - 1) / per : 0;
  if (x < tb) return RowBlock{x * per, min(T, (x + 1) * per)};
  const int nb = (L + per - 1) / per;
  const int f = (x - tb) / nb, j = x - tb - f * nb;
  const int s = T + f * L;
  return RowBlock{s + j * per, s + min(L, (j + 1) * per)};
}

// The tiles a workgroup visits along the other token axis: [0, a1) and [b0, b1) (the runs
// may overlap), so that the next tile is found without scanning the skipped ones.
struct TileRuns {
  int a1, b0, b1, n;
  // First visited tile >= t, or n when there is none.
  __device__ __forceinline__ int next(int t) const { return t < a1 ? t : (t < b1 ? max(t, b0) : n); }
};

// Workgroups are dispatched round-robin over the XCDs, each with its own L2. With `remap`,
// renumber the flattened grid so that each XCD runs one contiguous range of it: in the
// spatial branch the workgroups of one frame, which read the same key/value (or query)
// tiles, then share an L2. Joint attention keeps the dispatch order: there every
// workgroup of a head reads all of its tiles, and the XCDs working on the same head at the
// same time share them through the memory-side cache (renumbering spreads the XCDs over
// eight heads and costs ~7% in the key-stationary kernel). Returns (x, y, z).
constexpr int kXcds = 8;
__device__ __forceinline__ int3 xcd_grid_pos(bool remap) {
  if (!remap) return int3{(int)blockIdx.x, (int)blockIdx.y, (int)blockIdx.z};
  const int X = gridDim.x, Y = gridDim.y;
  const int G = X * Y * gridDim.z;
  const int i = blockIdx.x + X * (blockIdx.y + Y * blockIdx.z);
  const int q = G / kXcds, r = G % kXcds;
  const int xcd = i % kXcds, slot = i / kXcds;
  const int l = xcd < r ? xcd * (q + 1) + slot : r * (q + 1) + (xcd - r) * q + slot;
  return int3{l % X, (l / X) % Y, l / (X * Y)};
}

// Which (query, key) pairs attend. Key j of a sample is *valid* if j < N, it is not padded
// text (j >= T or j < tl) and key_mask keeps it. In joint attention every query sees every
// valid key. In the spatial branch (frame length L > 0) only video queries attend, to the
// valid text keys and to the valid keys of their own frame [T + f*L, T + (f+1)*L).
struct AttendRule {
  int N, T, tl, L;  // L = 0: joint attention
  const uint8_t* km;
  __device__ __forceinline__ int frame_start(int i) const { return T + ((i - T) / L) * L; }
  __device__ __forceinline__ bool key_valid(int j) const {
    bool ok = (j < N) & ((j >= T) | (j < tl));
    if (km) ok = ok & (km[min(j, N - 1)] != 0);  // unconditional clamped load
    return ok;
  }
  // The same for key j of the 64-key tile starting at k0, with the key mask of that tile
  // given as bits (bit i: key k0 + i kept; all ones without a mask), so that a per-element
  // test needs no load.
  __device__ __forceinline__ bool key_valid_bits(int j, int k0, unsigned long long bits) const {
    return (j < N) & ((j >= T) | (j < tl)) & (((bits >> (j - k0)) & 1ull) != 0);
  }
  // Lane `lane`'s byte of the key mask of tile kt (key kt*64 + lane, clamped to N-1), for
  // key_mask_bits; 1 without a mask (no load). Loaded a tile ahead of its use, so that its
  // wait is the one before the barrier at which that tile's copies have landed.
  __device__ __forceinline__ int key_mask_byte(int kt, int lane) const {
    return km ? (int)km[min(kt * kTileTok + lane, N - 1)] : 1;
  }
  // Key tiles a workgroup of queries [q0, q1) visits; uniform across the workgroup. Joint:
  // all but tiles of padded text only (when there is no key_mask). Spatial: the real text
  // tiles and the tiles of the frames its video queries lie in.
  __device__ __forceinline__ TileRuns key_tiles(int q0, int q1, int ntile) const {
    const int text_tiles = ((km ? T : tl) + kTileTok - 1) / kTileTok;
    if (L == 0) return km ? TileRuns{0, 0, ntile, ntile} : TileRuns{text_tiles, T / kTileTok, ntile, ntile};
    const int v0 = max(q0, T);
    if (v0 >= q1) return TileRuns{0, 0, 0, ntile};
    const int lo = frame_start(v0), hi = min(N, frame_start(q1 - 1) + L);
    return TileRuns{text_tiles, lo / kTileTok, (hi + kTileTok - 1) / kTileTok, ntile};
  }
  // Query tiles a workgroup of keys [k0, k1) visits (key-stationary kernels). Spatial: all
  // video query tiles if it holds real text keys, else the tiles of its keys' frames; never
  // a tile of text queries only.
  __device__ __forceinline__ TileRuns query_tiles(int k0, int k1, int ntile) const {
    if (L == 0) return TileRuns{0, 0, ntile, ntile};
    if (k0 < T && (km || k0 < tl)) return TileRuns{0, T / kTileTok, ntile, ntile};
    const int v0 = max(k0, T);
    if (v0 >= k1) return TileRuns{0, 0, 0, ntile};
    const int lo = frame_start(v0), hi = min(N, frame_start(k1 - 1) + L);
    return TileRuns{0, lo / kTileTok, (hi + kTileTok - 1) / kTileTok, ntile};
  }
};

// Spatial branch, query side: the keys query i attends to besides text, [lo, hi) (its own
// frame), and whether it attends to text at all (only video queries do).
struct QueryRange {
  int lo, hi;
  bool text;
  __device__ __forceinline__ bool ok(int j, int T) const { return j < T ? text : ((j >= lo) & (j < hi)); }
};
__device__ __forceinline__ QueryRange query_range(const AttendRule& r, int i) {
  if (r.L == 0 || i < r.T || i >= r.N) return QueryRange{0, 0, false};
  const int f0 = r.frame_start(i);
  return QueryRange{f0, f0 + r.L, true};
}
// Spatial branch, key side: the queries attending to key j, [lo, hi): every video query
// for a text key, the queries of its frame for a video key.
__device__ __forceinline__ int2 key_range(const AttendRule& r, int j) {
  if (r.L == 0) return int2{0, 0};
  if (j < r.T) return int2{r.T, r.N};
  const int f0 = r.frame_start(min(j, r.N - 1));
  return int2{f0, f0 + r.L};
}

// Kernel arguments. Token stride is H*D elements ([B, N, H, D] layout).
struct FwdArgs {
  const __bf16* q;
  const __bf16* k;
  const __bf16* vt;     // V as transposed token tiles
  const int32_t* text_len;
  const uint8_t* key_mask;
  __bf16* o;
  float* lse;
  int B, H, N, T, ntile;  // ntile = tiles of 64 tokens per (sample, head)
  int frame_len;          // 0: joint attention; > 0: spatial branch with frames of this many tokens
  float scale_log2;       // softmax scale times log2(e)
  // Joint attention: split tail over runs of tail_span key tiles. Per split workgroup row,
  // tail_part holds the unnormalised fp32 O ([tail_blocks][tail_chunks][256][D]), then the
  // exponent base m (log2 units) and the probability sum l ([tail_blocks][tail_chunks][256]).
  float* tail_part;
  int tail_blocks, tail_chunks, tail_span;
};

// Backward, key-stationary part: dK and dV.
struct DkdvArgs {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  const __bf16* dout;
  const __bf16* qt;     // Q as transposed token tiles
  const __bf16* dot;    // dO as transposed token tiles
  const float* lse2;    // LSE * log2(e), +inf for rows without keys and padding, [B, H, Npad]
  const float* dd;      // -D = -rowsum(dO o O), 0 on padding, [B, H, Npad]
  const int32_t* text_len;
  const uint8_t* key_mask;
  __bf16* dk;
  __bf16* dv;
  int B, H, N, T, ntile;
  int frame_len;        // 0: joint attention; > 0: spatial branch
  float scale;          // softmax scale
  float scale_log2;     // scale * log2(e)
  // Spatial branch, key blocks holding text keys (the first text_blocks): their video query
  // tiles are split into text_chunks runs of text_span tiles, one workgroup each, writing
  // fp32 partial dK, dV (scaled) to text_part, [2][text_chunks][B][H][text_blocks*256][D]
  // (dK partials, then dV). text_chunks = 1: no split, text_part unused.
  float* text_part;
  int text_blocks, text_chunks, text_span;
  // Joint attention: the tail_blocks items of the last, partial round of dispatch are each
  // split into tail_chunks workgroups over runs of tail_span query tiles, dispatched last,
  // writing fp32 partial dK, dV (scaled) to tail_part, [2][tail_blocks][tail_chunks][256][D].
  float* tail_part;
  int tail_blocks, tail_chunks, tail_span;
  // Joint attention with dQ fused in (dq_acc non-NULL): the workgroups of key blocks
  // [0, dq_blocks) also add their keys' share of dQ / scale, dS K, into the fp32
  // accumulator dq_acc ([B, N, H, D], zeroed by the launch) with atomics; the dQ pass adds
  // the share of the other keys. qt and dot are not read (transposed operands come from the
  // row-major tiles).
  float* dq_acc;
  int dq_blocks;
};

constexpr int kDkdvKeys = 256;  // keys per dK/dV workgroup

// Backward, query-stationary part: dQ.
struct DqArgs {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  const __bf16* dout;
  const __bf16* kt;     // K as transposed token tiles
  const float* lse2;
  const float* dd;
  const int32_t* text_len;
  const uint8_t* key_mask;
  __bf16* dq;
  int B, H, N, T, ntile;
  int frame_len;        // 0: joint attention; > 0: spatial branch
  float scale;
  float scale_log2;
  // Joint attention: split tail as for dK/dV, over runs of tail_span key tiles; fp32
  // partial dQ (scaled) in tail_part, [tail_blocks][tail_chunks][256][D].
  float* tail_part;
  int tail_blocks, tail_chunks, tail_span;
  // Completing a fused backward: only key tiles >= kt_min are visited, and dq_acc (fp32
  // [B, N, H, D], the other keys' dQ / scale) is added before scaling. kt_min = 0 and
  // dq_acc = NULL for the whole dQ.
  int kt_min;
  const float* dq_acc;
};

// Temporal branch: attention of each spatial position across the F frames. Video token
// (f, l) sits at T + f*L + l of the joint sequence. F <= 32: one wave handles G = 32/F
// positions; 32 < F <= kMaxTemporalFramesLong: one workgroup per position (frame blocks
// of 32), persistent over positions.
constexpr int kMaxTemporalFramesShort = 32;
constexpr int kMaxTemporalFramesLong = 144;
struct TemporalArgs {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  const __bf16* dout;   // backward only
  const uint8_t* key_mask;
  __bf16* o;            // forward output / backward dQ
  float* lse;           // forward output; backward: the forward's LSE (input)
  const __bf16* o_in;   // backward: the forward's O (for D = rowsum(dO o O))
  __bf16* dk;           // backward
  __bf16* dv;           // backward
  // Forward with the branch sum fused into the epilogue (sum_out non-NULL): also writes
  // sum_out = sum_a + sum_b + o for the video rows (a NULL input counts as zero).
  const __bf16* sum_a;
  const __bf16* sum_b;
  __bf16* sum_out;
  int B, H, N, T, F, L, G, npad;
  float scale;
  float scale_log2;
};

}  // namespace vcja

// Host-side launchers (defined in the .hip kernel files).
namespace vcja {
// Writes the transposed token tiles of x ([B, N, H, D]) into xt.
hipError_t launch_token_tiles(const __bf16* x, __bf16* xt, int B, int H, int N, int head_dim, hipStream_t s);
hipError_t launch_fwd(const FwdArgs& a, int head_dim, hipStream_t s);
hipError_t launch_bwd_prepare(const __bf16* o, const float* lse, const __bf16* dout, float* dd, float* lse2, int B,
                              int H, int N, int Npad, int head_dim, hipStream_t s);
hipError_t launch_bwd_dkdv(const DkdvArgs& a, int head_dim, hipStream_t s);
hipError_t launch_bwd_dq(const DqArgs& a, int head_dim, hipStream_t s);
// dq = bf16(scale * acc) over n elements (a fused backward whose key blocks all added their
// dQ share to the fp32 accumulator acc, [B, N, H, D] like dq). n a multiple of 4.
hipError_t launch_dq_from_acc(const float* acc, __bf16* dq, size_t n, float scale, hipStream_t s);
hipError_t launch_temporal_fwd(const TemporalArgs& a, int head_dim, hipStream_t s);
hipError_t launch_temporal_bwd(const TemporalArgs& a, int head_dim, hipStream_t s);
// Long clips (F > 32): persistent grid of at most `cus` workgroups. The backwards (both
// lengths) form -D and LSE*log2(e) themselves from o_in and lse.
hipError_t launch_temporal_long_fwd(const TemporalArgs& a, int head_dim, int cus, hipStream_t s);
hipError_t launch_temporal_long_bwd(const TemporalArgs& a, int head_dim, int cus, hipStream_t s);
// out = a + b + c over rows [0, rows) of every sample of [B, N, H, D] tensors (row_elems =
// H*D); each element summed in fp32 in that order and rounded once to bf16. A NULL input
// counts as zero; out may be one of the inputs.
hipError_t launch_branch_sum(const __bf16* a, const __bf16* b, const __bf16* c, __bf16* out, int B, int N, int rows,
                             int row_elems, hipStream_t s);
// Rows [0, T) of up to three [B, N, H, D] tensors set to zero and, if lse is given, their
// LSE ([B, H, N]) to -inf.
hipError_t launch_text_rows(__bf16* x0, __bf16* x1, __bf16* x2, float* lse, int B, int H, int N, int T, int head_dim,
                            hipStream_t s);
}  // namespace vcja
