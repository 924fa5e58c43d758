// decode_attn.hip -- gfx950 kernels and C ABI for single-query decode
// attention over a KV cache (MHA/GQA/MQA) and the per-step KV append.
//
// Kernels
//   kv_append_kernel       eqs. (6)-(7): bit-exact row copies per KV head,
//                          then len[b] += rows (Proposition 2's (d_k+d_v)*4
//                          bytes per row); T rows at once for multi-row steps.
//   decode_partial_kernel  eqs. (1)-(3) for all query heads of each GQA group
//                          at once, as per-visit partial states: every KV slab
//                          is read from HBM once and feeds all heads of its
//                          group (the group caching of the GQA section).
//                          Optionally fused with the append of the same step.
//                          The CAUSAL instances serve T query rows per head
//                          (a step that submits T positions); the direct form
//                          (one workgroup per single-chunk slab) writes the
//                          output itself, and in a fused step also advances
//                          len (the whole step in one launch).
//   decode_merge_kernel    combines each head's partials into its output row
//                          and resets the scheduling state.
//
// Work decomposition of decode_partial_kernel
//   A resident grid of 256-thread workgroups (4 waves) shares the slabs' rows:
//   most of each slab in ranges fixed in advance, proportional to the
//   lengths, the rest in small units handed out by per-slab counters (all
//   of it in ranges where a workgroup would hold too few units for the
//   hand-out to move work); a
//   workgroup's four waves share each 64-row turn of a segment, 16 rows
//   each (with one column block the waves' rows interleave in groups of
//   256/d rows, so the four waves' loads of one instruction cover 4 KB of
//   consecutive rows; see "Row-pair layout").  Each tile is two dense
//   products on the matrix cores
//   (v_mfma_f32_16x16x4_f32, fp32 in and out):
//     scores  S[16 rows x 16 heads] = K_tile[16 x d_k] . Q^T[d_k x 16]
//     update  O^T[d_v x 16 heads]  += V_tile^T[d_v x 16] . P[16 x 16 heads]
//   with the online (running reference / running sum) form of the softmax
//   between them, so the score vector never leaves registers.  Up to 16
//   query heads ride in one product's columns; groups of 17..32 heads use
//   two column blocks over the same K/V registers, larger groups several
//   head groups.
//   Scores are kept in base-2 units: q is pre-multiplied by scale*log2(e) and
//   exponentials are exp2, which is the hardware's native exponential.
//
// Register layouts of v_mfma_f32_16x16x4_f32 used below (lane = 0..63,
// i = lane % 16, k = lane / 16):
//   A operand (16 x 4):  lane holds A[i][k]
//   B operand (4 x 16):  lane holds B[k][i]
//   D result  (16 x 16): lane holds D[4k + r][i] in component r = 0..3
#include <hip/hip_runtime.h>

#include <cmath>
#include <algorithm>
#include <atomic>
#include <cstdint>
#include <cstdlib>

#include "decode_attn.h"

typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int kWave = 64;
constexpr int kWaves = 4;
constexpr int kThreads = kWave * kWaves;
constexpr int kTileRows = 16;                        // rows per MFMA tile
// Online softmax: each head's reference (the value its weights are
// exponentiated against, base-2 units) is raised only when a tile's maximum
// exceeds it by more than this, so a weight is at most 2^kLazyMax and the
// accumulators are rescaled only on such a jump (the result is the same
// softmax for any reference; the merge combines partials by their
// references).
constexpr float kLazyMax = 8.f;
constexpr int kHeadsPerBlock = 16;                   // heads per MFMA column block
constexpr int kMaxHeadBlocks = 2;                    // column blocks per workgroup
constexpr int kHeadsPerGroup = kHeadsPerBlock * kMaxHeadBlocks;
// Resident workgroups of the partial kernel: one per compute unit of the
// current device (hipDeviceAttributeMultiprocessorCount), at most this many
// -- the most CUs a gfx950 part has (MI355X: 256).  Workspace sizes are
// computed for this bound, so they hold on any device the library runs on.
constexpr int kMaxResident = 256;
// Register tiles per wave in the load ring of the partial kernel, which
// runs one wave per SIMD (all 512 registers of a lane).  One column block
// (<= 16 query rows per KV head): a three-tile ring keeps two tiles' loads in
// flight during each tile's products (two-tile rings at two waves per SIMD
// measured 2-4 % slower with fixed splits, and with the dynamic units below
// 10-30 % slower on long slabs).
// Two column blocks double the matrix work per tile: a four-tile ring (three
// tiles in flight), with both blocks' score chains, softmax updates and
// weighted sums issued side by side, is 6 % faster on MQA than a two-tile
// ring at two waves per SIMD, 7 % faster than a three-tile ring.  A tile of
// d_k = d_v = 256 holds 128 registers per lane: such head sizes take a
// two-tile ring.  The direct form of one column block (every slab a single
// chunk, one workgroup per slab) runs instead at two waves per SIMD with a
// two-tile ring (the W = 2 instances): two co-resident workgroups overlap
// one's start and drain with the other's streaming, 3.5-7.5 % faster on
// short caches (n <= 768) of many slabs, and 4-10 % faster than the
// persistent form on batches of at least 2048 slabs of up to 4608 rows.
// Tiles in the ring of the persistent (one wave per SIMD) instances; the
// host's scheduling unit is one turn of it.
__host__ __device__ constexpr int ring_tiles(int nb, int dk, int dv) {
  return dk + dv > 256 ? 2 : (nb == 2 ? 4 : 3);
}
template <int NB, int DK, int DV>
constexpr int kRing = ring_tiles(NB, DK, DV);
// q of the visit's heads (the B operand of the score products) is held in
// registers for the whole visit where they fit (NB * d_k / 4 per lane, one
// wave per SIMD), else re-read from LDS for every tile.  Two column blocks
// at d_k = 256 would need 128 registers for it.
template <int NB, int DK>
constexpr bool kPinQ = NB * DK <= 256;
// A segment (chunk_rows) is the most rows a workgroup reads in one go from
// its static range, a multiple of twelve 16-row tiles per wave (whole turns
// of every ring); with no static share (single-chunk caches, very large
// batches) it is also the unit handed out dynamically.
constexpr int kChunkQuantum = 12 * kTileRows * kWaves;
static_assert(12 % 2 == 0 && 12 % 3 == 0 && 12 % 4 == 0, "chunks are whole turns of every ring");
constexpr int kDefaultChunkRows = 768;
// Many short slabs: with at least kDirectMinSlabs slabs (four rounds of the
// 512 two-wave workgroup slots of 256 CUs) of at most kDirectMaxRows rows,
// one column block and d_k + d_v <= 256, the library takes each slab whole
// as one segment, so that the direct form runs: one workgroup per slab, two
// per CU, the hardware dispatcher balancing the slabs and no merge launch.
// (Measured on uniform and ragged lengths; with fewer slabs, ragged lengths
// leave the last round's long slabs alone on the chip.)
constexpr int64_t kDirectMinSlabs = 2048;
constexpr int kDirectMaxRows = 6 * kChunkQuantum;
// Visit slots per slab for dynamic visits, in units of the even share of
// resident workgroups per slab.
constexpr int kVisitSlack = 4;
// Static share of each slab's rows, in sixteenths: the first
// floor(14/16 * rows / Cd) units of Cd rows (one turn of the tile ring) of
// every slab are divided among the workgroups in advance, the rest is handed
// out dynamically one unit at a time.  With at least two slabs per resident
// workgroup (one column block) the share is 16/16: every slab is wholly
// static, ceil(rows / Cd) units, and nothing is searched for or claimed.
// Batches of more than kMaxStaticSeqs sequences would make the
// per-workgroup prefix sums long: they are scheduled dynamically only.
constexpr int kStaticDen = 16;
constexpr int kStaticNum = 14;
constexpr int kMaxStaticSeqs = 256;
// The dynamic share pays only where each workgroup holds enough units for it
// to move: a workgroup commits two to three units ahead, so with fewer than
// kDynamicMinUnits units per resident workgroup (counted at n_max rows per
// slab) every slab is wholly static instead -- no claims, no per-unit
// barriers, no dynamic visits.  (Measured: MQA 16384 rows 2.7 % faster, short
// and ragged batches of 10-22 units per workgroup 5-10 % faster, batches of
// 43 units per workgroup level to 2 % slower, longer ones unchanged.)  The
// environment variable DECODE_ATTN_DYNAMIC_MIN_UNITS overrides the bound (0:
// the static share wherever it applied before; for tests and tuning).
constexpr int kDynamicMinUnits = 32;
// A batch of fewer than kTwoWaveMaxUnits one-wave units per CU of the
// largest grid (counted at n_max rows per slab) runs, with one column block
// and a wholly static plan, as whole-slab ranges at two workgroups per CU
// whatever its slabs' length: one workgroup's visit set-up and drain overlap
// the other's streaming.  Measured on batches of 1-4 sequences of 16-64k
// rows (8-16 units per workgroup): 5.7-8.4 % faster; at 22 units per
// workgroup (MHA 8 x 32 heads x 4112 rows, GQA-4 16 x 8192 rows) 0.1-0.4 %
// slower, so those keep one workgroup per CU.
constexpr int kTwoWaveMaxUnits = 16;
constexpr int64_t kMaxSlabs = 1 << 20;
constexpr int kMaxQueryRows = 4096;                  // T of a multi-row decode
// Each slab's scheduling word, {dynamic units taken (low half), dynamic
// visits opened (high half)}, has a 128-byte line of its own, so atomics on
// different slabs' words never serialize on the same line.
constexpr int kCounterStride = 32;
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ f4 mfma_16x16x4(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) {
  return __builtin_amdgcn_exp2f(x);  // v_exp_f32; exp2(-inf) = 0
}

__device__ __forceinline__ f4 load4(const float* p) {
  return *reinterpret_cast<const f4*>(p);
}

// K/V rows are read once per decode.  A V load instruction consumes whole
// 128-byte lines (16 lanes x 16 bytes of one row), so V streams past the
// caches; a K load instruction reads half of each of 16 lines and the next
// one the other half, so K loads keep the default policy and the second
// half can be served from cache (measured: 2 % faster on long contexts, 5 %
// on MQA, than streaming K too).
__device__ __forceinline__ f4 load4_stream(const float* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const f4*>(p));
}

// Reductions over the four 16-lane row groups of a wave (lanes i, i+16,
// i+32, i+48 hold the same head in the score layout).  permlane16_swap(x, x)
// returns the row pairs (r0,r0,r2,r2) and (r1,r1,r3,r3), permlane32_swap the
// halves (lo,lo) and (hi,hi): two VALU swaps instead of two LDS shuffles.
__device__ __forceinline__ float max_over_row_groups(float x) {
  const unsigned u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float m = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const unsigned v = __float_as_uint(m);
  const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ float sum_over_row_groups(float x) {
  const unsigned u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float m = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const unsigned v = __float_as_uint(m);
  const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

__device__ __forceinline__ int rows_used(int32_t len_b, int n_max) {
  return len_b < 0 ? 0 : (len_b > n_max ? n_max : len_b);
}

// With a fused append of T rows, the decode of sequence b also covers the
// appended rows len[b] .. len[b]+T-1 that fit in the cache.
__device__ __forceinline__ bool appends(bool app, int32_t len_b, int n_max) {
  return app && len_b >= 0 && len_b < n_max;
}

__device__ __forceinline__ int appended_rows(bool app, int32_t len_b, int n_max, int T) {
  return appends(app, len_b, n_max) ? min(T, n_max - len_b) : 0;
}

__device__ __forceinline__ int decode_rows(int32_t len_b, int n_max, bool app, int T) {
  return appends(app, len_b, n_max) ? len_b + appended_rows(app, len_b, n_max, T)
                                    : rows_used(len_b, n_max);
}

// ---------------------------------------------------------------------------
// KV append of T rows.  One workgroup per sequence; every thread reads len[b]
// before the barrier, thread 0 writes it after, so no thread can see the new
// value.  Rows r = 0..T-1 land at len[b] + r as long as they fit (the
// single-row append applied T times).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void kv_append_kernel(
    float* __restrict__ K, float* __restrict__ V,
    const float* __restrict__ k_new, const float* __restrict__ v_new,
    int32_t* __restrict__ len, int h_kv, int n_max, int d_k, int d_v, int T) {
  const int b = blockIdx.x;
  const int32_t t = len[b];
  const int cnt = (t >= 0 && t < n_max) ? min(T, n_max - t) : 0;
  if (cnt > 0) {
    const int ck = d_k / 4, cv = d_v / 4;            // 16-byte chunks per row
    const int per_row = ck + cv;
    const int per_head = cnt * per_row;
    const int total = h_kv * per_head;
    for (int c = threadIdx.x; c < total; c += blockDim.x) {
      const int g = c / per_head;
      const int rem = c - g * per_head;
      const int r = rem / per_row;
      const int w = rem - r * per_row;
      const int64_t slab = (int64_t)b * h_kv + g;
      const int64_t src_row = slab * T + r;
      const int64_t dst_row = slab * n_max + t + r;
      if (w < ck) {
        const u4* src = reinterpret_cast<const u4*>(k_new + src_row * d_k) + w;
        u4* dst = reinterpret_cast<u4*>(K + dst_row * d_k) + w;
        *dst = *src;
      } else {
        const int wv = w - ck;
        const u4* src = reinterpret_cast<const u4*>(v_new + src_row * d_v) + wv;
        u4* dst = reinterpret_cast<u4*>(V + dst_row * d_v) + wv;
        *dst = *src;
      }
    }
  }
  __syncthreads();
  if (cnt > 0 && threadIdx.x == 0) len[b] = t + cnt;
}

// ---------------------------------------------------------------------------
// Register tiles and tile processing of the decode.
// ---------------------------------------------------------------------------
template <int DK, int DV, int NB>
struct Tile {
  f4 k[DK / 16];          // K rows: lane (i,k) holds row i, dims 16t+4k..+3
  f4 v[4][DV / 64];       // V rows: lane (i,k) holds row 4k+rho, dims 64c+4i..+3
};

// Where a tile's rows live: the slab, except rows new_lo .. new_lo+new_cnt-1
// (the rows a fused append adds; new_cnt = 0 if none), which are read from the
// incoming k_new / v_new rows.  new_row is new_lo when exactly one row is
// added, else -1.  Rows [0, fast_end) are plain slab rows.
struct RowSource {
  const float* __restrict__ Ks;
  const float* __restrict__ Vs;
  const float* __restrict__ k_new_rows;
  const float* __restrict__ v_new_rows;
  int new_lo;
  int new_cnt;
  int new_row;
  int fast_end;
  uint32_t k_lane;          // byte offset of lane (i,k) in a K tile: i*d_k + 4k floats
  uint32_t v_lane;          // byte offset of lane (i,k) in a V tile: 4k*d_v + 4i floats
  // Row-pair layout only (see below).
  int wave;                 // this wave's index in the workgroup
  int first_off, max_off;   // offsets of the wave's first and last tile row from its turn
  uint32_t kw_lane;         // LDS byte offset this lane writes K to (plus a per-load constant)
  uint32_t kr_lane;         // LDS byte offset this lane reads K from (plus 64 bytes per t)
  int rowoff[4];            // offset from the turn of the row score component r stands for
};

// ROWS: a fused append may add several rows (multi-row steps); otherwise at
// most one, which keeps the redirect a single comparison.
template <int DK, int DV, int NB, bool ROWS>
__device__ __forceinline__ void load_tile(Tile<DK, DV, NB>& T, const RowSource& src,
                                          int row0, int last_row, int i, int k) {
  if (row0 + kTileRows <= src.fast_end) {
    // Interior tile: one wave-uniform row base and a fixed per-lane offset,
    // so every load is scalar base + lane offset + immediate (no per-tile
    // address arithmetic on the vector ALUs).
    const char* kb = reinterpret_cast<const char*>(src.Ks + (int64_t)row0 * DK);
    const char* vb = reinterpret_cast<const char*>(src.Vs + (int64_t)row0 * DV);
#pragma unroll
    for (int t = 0; t < DK / 16; ++t)
      T.k[t] = load4(reinterpret_cast<const float*>(kb + src.k_lane) + 16 * t);
#pragma unroll
    for (int rho = 0; rho < 4; ++rho)
#pragma unroll
      for (int c = 0; c < DV / 64; ++c)
        T.v[rho][c] =
            load4_stream(reinterpret_cast<const float*>(vb + src.v_lane) + rho * DV + 64 * c);
    return;
  }
  // The slab's last tile(s): rows past the end clamp to the last row, and
  // the rows a fused append adds come from k_new / v_new.  (The lane indices
  // are made opaque here so that this rarely taken path's per-lane addresses
  // are formed inside it, not hoisted out of the tile loop into registers.)
  asm volatile("" : "+v"(i), "+v"(k));
  const int rk = min(row0 + i, last_row);
  const float* kp;
  if constexpr (ROWS)
    kp = (unsigned)(rk - src.new_lo) < (unsigned)src.new_cnt
             ? src.k_new_rows + (rk - src.new_lo) * DK
             : src.Ks + (int64_t)rk * DK;
  else
    kp = rk == src.new_row ? src.k_new_rows : src.Ks + (int64_t)rk * DK;
#pragma unroll
  for (int t = 0; t < DK / 16; ++t) T.k[t] = load4(kp + 16 * t + 4 * k);
#pragma unroll
  for (int rho = 0; rho < 4; ++rho) {
    const int rv = min(row0 + 4 * k + rho, last_row);
    const float* vp;
    if constexpr (ROWS)
      vp = (unsigned)(rv - src.new_lo) < (unsigned)src.new_cnt
               ? src.v_new_rows + (rv - src.new_lo) * DV
               : src.Vs + (int64_t)rv * DV;
    else
      vp = rv == src.new_row ? src.v_new_rows : src.Vs + (int64_t)rv * DV;
#pragma unroll
    for (int c = 0; c < DV / 64; ++c) T.v[rho][c] = load4_stream(vp + 64 * c + 4 * i);
  }
}

// ---------------------------------------------------------------------------
// Row-pair layout (one column block, one wave per SIMD).  Each 16-byte load
// instruction of a wave reads 1 KB of consecutive cache rows -- 256/d rows of
// a d-wide tensor (2 rows at d = 128) -- instead of 64 bytes from each of 16
// rows, so that every instruction covers whole 128-byte lines of one
// contiguous run.  The MFMA operands need 16 rows spread over the lanes, so:
//   V: two (d = 128) or four (d = 256) loaded registers are regrouped with
//      v_permlane16_swap / v_permlane32_swap into the A-operand layout of the
//      update product (lane (i,k): one row per lane-row k, dims 4i..4i+3 of a
//      64-dim block); at d = 64 a load already is that layout.  This fixes
//      which tile row each score row must be: update group rho takes tile rows
//      upd_row(rho, k), k = 0..3, so score row 4k + rho is tile row
//      upd_row(rho, k).
//   K: written to a wave-private LDS tile whose slots are the score rows (slot
//      4k + rho holds tile row upd_row(rho, k)), then read back in the A-operand
//      layout of the score product (lane (i,k) reads slot i, dims
//      16t + 4k..+3).  A slot is d_k + 4 floats wide, so the 8 lanes of a
//      128-bit LDS access hit 8 different bank groups on both sides.
// With kAdjacent the four waves of a workgroup read neighbouring row groups:
// a wave's tile rows interleave with the other waves' across the 64-row turn
// (4 KB contiguous per workgroup and load instruction) instead of being 16
// consecutive rows.
// ---------------------------------------------------------------------------
template <int NB, int W>
constexpr bool kPairs = NB == 1 && W == 1;
// (K and V must cover the same rows per load for the interleaved order.)
template <int DK, int DV>
constexpr bool kAdjacent = DK == DV;

// Offset of tile row q (0..15) of wave w from the first row of its turn; rpl
// rows per load instruction.
template <int RPL, bool ADJ>
__device__ __forceinline__ int tile_row_off(int q, int w) {
  if constexpr (ADJ) return 4 * RPL * (q / RPL) + RPL * w + q % RPL;
  else return 16 * w + q;
}

// Tile row of lane-row k in update group rho (the row order the V regrouping
// produces).
template <int DV>
__host__ __device__ constexpr int upd_row(int rho, int k) {
  return DV == 128 ? 4 * rho + 2 * (k & 1) + (k >> 1) : 4 * rho + k;
}

// LDS slot (= score row) of tile row q: the inverse of upd_row.
template <int DV>
__host__ __device__ constexpr int slot_of_row(int q) {
  return DV == 128 ? 4 * (((q >> 1) & 1) + 2 * (q & 1)) + (q >> 2) : 4 * (q & 3) + (q >> 2);
}

// Bytes per LDS slot of the K tile.
template <int DK>
constexpr int kKSlot = 4 * DK + 16;

__device__ __forceinline__ void swap16(f4& a, f4& b) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a[e]), __float_as_uint(b[e]),
                                                    false, false);
    a[e] = __uint_as_float(r[0]);
    b[e] = __uint_as_float(r[1]);
  }
}

__device__ __forceinline__ void swap32(f4& a, f4& b) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a[e]), __float_as_uint(b[e]),
                                                    false, false);
    a[e] = __uint_as_float(r[0]);
    b[e] = __uint_as_float(r[1]);
  }
}

// Per-lane constants of the row-pair layout for wave w, lane (i, k).
template <int DK, int DV>
__device__ __forceinline__ void pair_lane_setup(RowSource& src, int w, int i, int k) {
  constexpr bool ADJ = kAdjacent<DK, DV>;
  constexpr int RK = 256 / DK, RV = 256 / DV;
  const int lane = i + 16 * k;
  src.wave = w;
  // (for ADJ, d_k = d_v: one rows-per-load for both)
  src.first_off = tile_row_off<RV, ADJ>(0, w);
  src.max_off = tile_row_off<RV, ADJ>(15, w);
  src.k_lane = (uint32_t)(tile_row_off<RK, ADJ>(0, w) * DK * 4 + 16 * lane);
  src.v_lane = (uint32_t)(tile_row_off<RV, ADJ>(0, w) * DV * 4 + 16 * lane);
  const int jk = lane / (DK / 4), ck = lane % (DK / 4);
  src.kw_lane = (uint32_t)(slot_of_row<DV>(jk) * kKSlot<DK> + 16 * ck);
  src.kr_lane = (uint32_t)(i * kKSlot<DK> + 16 * k);
#pragma unroll
  for (int r = 0; r < 4; ++r) src.rowoff[r] = tile_row_off<RV, ADJ>(upd_row<DV>(r, k), w);
}

// Loads of one tile in the row-pair layout: load m of K covers tile rows
// RK*m .. RK*m+RK-1 (lane: row RK*m + lane/(d_k/4), 16-byte piece lane %
// (d_k/4)), likewise V.  row0 = the turn's first row + first_off.
template <int DK, int DV, int NB, bool ROWS>
__device__ __forceinline__ void load_tile_pairs(Tile<DK, DV, NB>& T, const RowSource& src,
                                                int row0, int last_row, int lane) {
  constexpr bool ADJ = kAdjacent<DK, DV>;
  constexpr int RK = 256 / DK, RV = 256 / DV;
  constexpr int kStep = ADJ ? 4096 : 1024;            // bytes between a wave's loads
  const int tb = row0 - src.first_off;
  if (tb + src.max_off < src.fast_end) {
    const char* kb = reinterpret_cast<const char*>(src.Ks + (int64_t)tb * DK) + src.k_lane;
    const char* vb = reinterpret_cast<const char*>(src.Vs + (int64_t)tb * DV) + src.v_lane;
#pragma unroll
    for (int m = 0; m < DK / 16; ++m)
      T.k[m] = load4_stream(reinterpret_cast<const float*>(kb + m * kStep));
#pragma unroll
    for (int m = 0; m < DV / 16; ++m)
      T.v[m / (DV / 64)][m % (DV / 64)] =
          load4_stream(reinterpret_cast<const float*>(vb + m * kStep));
    return;
  }
  // Rows past the end clamp to the last row (and to row 0 for the dummy
  // loads past a visit's end); appended rows come from k_new / v_new.
  auto source = [&](const float* base, const float* nbase, int D, int row) -> const float* {
    row = max(0, min(row, last_row));
    if constexpr (ROWS) {
      if ((unsigned)(row - src.new_lo) < (unsigned)src.new_cnt)
        return nbase + (int64_t)(row - src.new_lo) * D;
    } else {
      if (row == src.new_row) return nbase;
    }
    return base + (int64_t)row * D;
  };
  const int jk = lane / (DK / 4), ck = lane % (DK / 4);
#pragma unroll
  for (int m = 0; m < DK / 16; ++m) {
    const int row = tb + tile_row_off<RK, ADJ>(RK * m + jk, src.wave);
    T.k[m] = load4_stream(source(src.Ks, src.k_new_rows, DK, row) + 4 * ck);
  }
  const int jv = lane / (DV / 4), cv = lane % (DV / 4);
#pragma unroll
  for (int m = 0; m < DV / 16; ++m) {
    const int row = tb + tile_row_off<RV, ADJ>(RV * m + jv, src.wave);
    T.v[m / (DV / 64)][m % (DV / 64)] = load4_stream(source(src.Vs, src.v_new_rows, DV, row) + 4 * cv);
  }
}

// One tile in the row-pair layout, one column block: K through the wave's LDS
// slots into the score operand layout, V regrouped into the update operand
// layout, then the same products and online softmax as process_tile.
template <int DK, int DV, int NB, bool CAUSAL, bool PINQ>
__device__ __forceinline__ void process_tile_pairs(const Tile<DK, DV, NB>& T, int row0,
                                                   const int (&lim)[NB], const RowSource& src,
                                                   int lane, char* __restrict__ wk,
                                                   const f4 (*__restrict__ sh_q)[DK / 16][kWave],
                                                   const f4 (&qr)[NB][DK / 16],
                                                   float (&m_run)[NB], float (&l_run)[NB],
                                                   f4 (&acc)[NB][DV / 64][4]) {
  static_assert(NB == 1, "row-pair layout: one column block");
  constexpr int RK = 256 / DK;
  if constexpr (!PINQ) asm volatile("" ::: "memory");
  // K: tile rows to their score-row slots, then the operand layout.
#pragma unroll
  for (int m = 0; m < DK / 16; ++m)
    *reinterpret_cast<f4*>(wk + src.kw_lane + slot_of_row<DV>(RK * m) * kKSlot<DK>) = T.k[m];
  __builtin_amdgcn_wave_barrier();
  f4 kt[DK / 16];
#pragma unroll
  for (int t = 0; t < DK / 16; ++t)
    kt[t] = *reinterpret_cast<const f4*>(wk + src.kr_lane + 64 * t);
  __builtin_amdgcn_wave_barrier();
  // V: the update operand of group rho, block c.
  f4 va[4][DV / 64];
#pragma unroll
  for (int rho = 0; rho < 4; ++rho)
#pragma unroll
    for (int c = 0; c < DV / 64; ++c) va[rho][c] = T.v[rho][c];
  if constexpr (DV == 128) {
#pragma unroll
    for (int rho = 0; rho < 4; ++rho) swap16(va[rho][0], va[rho][1]);
  } else if constexpr (DV == 256) {
#pragma unroll
    for (int rho = 0; rho < 4; ++rho) {
      swap32(va[rho][0], va[rho][2]);
      swap32(va[rho][1], va[rho][3]);
      swap16(va[rho][0], va[rho][1]);
      swap16(va[rho][2], va[rho][3]);
    }
  }
  auto Q = [&](int t) -> f4 {
    if constexpr (PINQ) return qr[0][t];
    else return sh_q[0][t][lane];
  };
  f4 s0 = f4{0.f, 0.f, 0.f, 0.f}, s1 = s0;
#pragma unroll
  for (int t = 0; t < DK / 16; t += 2) {
    const f4 q0 = Q(t), q1 = Q(t + 1);
    s0 = mfma_16x16x4(kt[t].x, q0.x, s0);
    s1 = mfma_16x16x4(kt[t + 1].x, q1.x, s1);
    s0 = mfma_16x16x4(kt[t].y, q0.y, s0);
    s1 = mfma_16x16x4(kt[t + 1].y, q1.y, s1);
    s0 = mfma_16x16x4(kt[t].z, q0.z, s0);
    s1 = mfma_16x16x4(kt[t + 1].z, q1.z, s1);
    s0 = mfma_16x16x4(kt[t].w, q0.w, s0);
    s1 = mfma_16x16x4(kt[t + 1].w, q1.w, s1);
  }
  f4 s = s0 + s1;
  const int tb = row0 - src.first_off;
  if (CAUSAL || tb + src.max_off > lim[0]) {
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (tb + src.rowoff[r] > lim[0]) s[r] = -INFINITY;
  }
  const float tmax = max_over_row_groups(fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3])));
  const bool bump = tmax > m_run[0] + kLazyMax;
  if (__any(bump)) {
    const float m_new = bump ? tmax : m_run[0];
    float m_ref = m_new;
    if constexpr (CAUSAL) m_ref = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = fast_exp2(m_run[0] - m_ref);
    l_run[0] *= alpha;
#pragma unroll
    for (int c = 0; c < DV / 64; ++c)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[0][c][e] *= alpha;
    m_run[0] = m_new;
  }
  float m_ref = m_run[0];
  if constexpr (CAUSAL) m_ref = m_ref == -INFINITY ? 0.f : m_ref;
  f4 pr;
  pr[0] = fast_exp2(s[0] - m_ref);
  pr[1] = fast_exp2(s[1] - m_ref);
  pr[2] = fast_exp2(s[2] - m_ref);
  pr[3] = fast_exp2(s[3] - m_ref);
  l_run[0] += (pr[0] + pr[1]) + (pr[2] + pr[3]);
#pragma unroll
  for (int rho = 0; rho < 4; ++rho)
#pragma unroll
    for (int c = 0; c < DV / 64; ++c) {
      acc[0][c][0] = mfma_16x16x4(va[rho][c].x, pr[rho], acc[0][c][0]);
      acc[0][c][1] = mfma_16x16x4(va[rho][c].y, pr[rho], acc[0][c][1]);
      acc[0][c][2] = mfma_16x16x4(va[rho][c].z, pr[rho], acc[0][c][2]);
      acc[0][c][3] = mfma_16x16x4(va[rho][c].w, pr[rho], acc[0][c][3]);
    }
}

// One 16-row tile for NB column blocks of query heads: scores on the matrix
// cores, online softmax update, weighted-sum update on the matrix cores.
template <int DK, int DV, int NB, bool CAUSAL, bool PINQ>
__device__ __forceinline__ void process_tile(const Tile<DK, DV, NB>& T, int row0,
                                             const int (&lim)[NB], int k, int lane,
                                             const f4 (*__restrict__ sh_q)[DK / 16][kWave],
                                             const f4 (&qr)[NB][DK / 16],
                                             float (&m_run)[NB], float (&l_run)[NB],
                                             f4 (&acc)[NB][DV / 64][4]) {
  // Unpinned, q is re-read from LDS for every tile: the empty asm keeps the
  // compiler from hoisting those reads out of the tile loop.
  if constexpr (!PINQ) asm volatile("" ::: "memory");
  auto Q = [&](int nb, int t) -> f4 {
    if constexpr (PINQ) return qr[nb][t];
    else return sh_q[nb][t][lane];
  };
  if constexpr (NB == 2) {
    // Both column blocks in step: their score chains (four independent
    // accumulators sharing each K operand), then both softmax updates, then
    // both weighted sums sharing each V operand.
    f4 sa0 = f4{0.f, 0.f, 0.f, 0.f}, sa1 = sa0, sb0 = sa0, sb1 = sa0;
#pragma unroll
    for (int t = 0; t < DK / 16; t += 2) {
      const f4 qa0 = Q(0, t), qa1 = Q(0, t + 1);
      const f4 qb0 = Q(1, t), qb1 = Q(1, t + 1);
      sa0 = mfma_16x16x4(T.k[t].x, qa0.x, sa0);
      sb0 = mfma_16x16x4(T.k[t].x, qb0.x, sb0);
      sa1 = mfma_16x16x4(T.k[t + 1].x, qa1.x, sa1);
      sb1 = mfma_16x16x4(T.k[t + 1].x, qb1.x, sb1);
      sa0 = mfma_16x16x4(T.k[t].y, qa0.y, sa0);
      sb0 = mfma_16x16x4(T.k[t].y, qb0.y, sb0);
      sa1 = mfma_16x16x4(T.k[t + 1].y, qa1.y, sa1);
      sb1 = mfma_16x16x4(T.k[t + 1].y, qb1.y, sb1);
      sa0 = mfma_16x16x4(T.k[t].z, qa0.z, sa0);
      sb0 = mfma_16x16x4(T.k[t].z, qb0.z, sb0);
      sa1 = mfma_16x16x4(T.k[t + 1].z, qa1.z, sa1);
      sb1 = mfma_16x16x4(T.k[t + 1].z, qb1.z, sb1);
      sa0 = mfma_16x16x4(T.k[t].w, qa0.w, sa0);
      sb0 = mfma_16x16x4(T.k[t].w, qb0.w, sb0);
      sa1 = mfma_16x16x4(T.k[t + 1].w, qa1.w, sa1);
      sb1 = mfma_16x16x4(T.k[t + 1].w, qb1.w, sb1);
    }
    f4 sc[2] = {sa0 + sa1, sb0 + sb1};
    f4 pr[2];
    float tmax[2];
    bool bump[2];
    // Rows past the last row a column sees take no weight (only a slab's
    // last tile has any, unless the columns are causal).
    const bool mask = CAUSAL || row0 + kTileRows - 1 > lim[0];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      if (mask) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (row0 + 4 * k + r > lim[nb]) sc[nb][r] = -INFINITY;
      }
      tmax[nb] =
          max_over_row_groups(fmaxf(fmaxf(sc[nb][0], sc[nb][1]), fmaxf(sc[nb][2], sc[nb][3])));
      bump[nb] = tmax[nb] > m_run[nb] + kLazyMax;
    }
    // A reference moves (rarely): rescale the sums of the heads it moves for.
    if (__any(bump[0] || bump[1])) {
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const float m_new = bump[nb] ? tmax[nb] : m_run[nb];
        float m_ref = m_new;
        if constexpr (CAUSAL) m_ref = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = fast_exp2(m_run[nb] - m_ref);
        l_run[nb] *= alpha;
#pragma unroll
        for (int c = 0; c < DV / 64; ++c)
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[nb][c][e] *= alpha;
        m_run[nb] = m_new;
      }
    }
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      // A causal column may have seen no row yet (reference -inf):
      // exponentiate against 0 then, so every weight is 0 instead of NaN.
      float m_ref = m_run[nb];
      if constexpr (CAUSAL) m_ref = m_ref == -INFINITY ? 0.f : m_ref;
      pr[nb][0] = fast_exp2(sc[nb][0] - m_ref);
      pr[nb][1] = fast_exp2(sc[nb][1] - m_ref);
      pr[nb][2] = fast_exp2(sc[nb][2] - m_ref);
      pr[nb][3] = fast_exp2(sc[nb][3] - m_ref);
      l_run[nb] += (pr[nb][0] + pr[nb][1]) + (pr[nb][2] + pr[nb][3]);
    }
#pragma unroll
    for (int rho = 0; rho < 4; ++rho)
#pragma unroll
      for (int c = 0; c < DV / 64; ++c) {
        acc[0][c][0] = mfma_16x16x4(T.v[rho][c].x, pr[0][rho], acc[0][c][0]);
        acc[1][c][0] = mfma_16x16x4(T.v[rho][c].x, pr[1][rho], acc[1][c][0]);
        acc[0][c][1] = mfma_16x16x4(T.v[rho][c].y, pr[0][rho], acc[0][c][1]);
        acc[1][c][1] = mfma_16x16x4(T.v[rho][c].y, pr[1][rho], acc[1][c][1]);
        acc[0][c][2] = mfma_16x16x4(T.v[rho][c].z, pr[0][rho], acc[0][c][2]);
        acc[1][c][2] = mfma_16x16x4(T.v[rho][c].z, pr[1][rho], acc[1][c][2]);
        acc[0][c][3] = mfma_16x16x4(T.v[rho][c].w, pr[0][rho], acc[0][c][3]);
        acc[1][c][3] = mfma_16x16x4(T.v[rho][c].w, pr[1][rho], acc[1][c][3]);
      }
    return;
  }
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    // Step I: s[row 4k+r][head i] for the tile's 16 rows (two independent
    // accumulation chains over the d_k/4 steps, added at the end).  q is
    // fetched pair by pair (from LDS unless pinned), so at two waves per SIMD
    // only four of its registers are live at a time.
    f4 s0 = f4{0.f, 0.f, 0.f, 0.f}, s1 = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < DK / 16; t += 2) {
      const f4 qa = Q(nb, t), qc = Q(nb, t + 1);
      s0 = mfma_16x16x4(T.k[t].x, qa.x, s0);
      s1 = mfma_16x16x4(T.k[t + 1].x, qc.x, s1);
      s0 = mfma_16x16x4(T.k[t].y, qa.y, s0);
      s1 = mfma_16x16x4(T.k[t + 1].y, qc.y, s1);
      s0 = mfma_16x16x4(T.k[t].z, qa.z, s0);
      s1 = mfma_16x16x4(T.k[t + 1].z, qc.z, s1);
      s0 = mfma_16x16x4(T.k[t].w, qa.w, s0);
      s1 = mfma_16x16x4(T.k[t + 1].w, qc.w, s1);
    }
    f4 s = s0 + s1;
    // Rows past the last row this lane's column sees take no weight (only a
    // slab's last tile has any, unless the columns are causal).
    if (CAUSAL || row0 + kTileRows - 1 > lim[nb]) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (row0 + 4 * k + r > lim[nb]) s[r] = -INFINITY;
    }

    // Step II, online: the tile's max over the 4 row groups of head i; the
    // head's reference moves only on a jump above kLazyMax, and then (rarely)
    // the sums are rescaled.
    const float tmax = max_over_row_groups(fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3])));
    const bool bump = tmax > m_run[nb] + kLazyMax;
    if (__any(bump)) {
      const float m_new = bump ? tmax : m_run[nb];
      float m_ref = m_new;
      if constexpr (CAUSAL) m_ref = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = fast_exp2(m_run[nb] - m_ref);
      l_run[nb] *= alpha;
#pragma unroll
      for (int c = 0; c < DV / 64; ++c)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[nb][c][e] *= alpha;
      m_run[nb] = m_new;
    }
    // A causal column may have seen no row yet (reference -inf): exponentiate
    // against 0 then, so every weight is 0 instead of NaN.
    float m_ref = m_run[nb];
    if constexpr (CAUSAL) m_ref = m_ref == -INFINITY ? 0.f : m_ref;
    f4 pr;
    pr[0] = fast_exp2(s[0] - m_ref);
    pr[1] = fast_exp2(s[1] - m_ref);
    pr[2] = fast_exp2(s[2] - m_ref);
    pr[3] = fast_exp2(s[3] - m_ref);
    l_run[nb] += (pr[0] + pr[1]) + (pr[2] + pr[3]);

    // Step III: acc += V_tile^T . P over rows {rho, 4+rho, 8+rho, 12+rho}.
#pragma unroll
    for (int rho = 0; rho < 4; ++rho)
#pragma unroll
      for (int c = 0; c < DV / 64; ++c) {
        acc[nb][c][0] = mfma_16x16x4(T.v[rho][c].x, pr[rho], acc[nb][c][0]);
        acc[nb][c][1] = mfma_16x16x4(T.v[rho][c].y, pr[rho], acc[nb][c][1]);
        acc[nb][c][2] = mfma_16x16x4(T.v[rho][c].z, pr[rho], acc[nb][c][2]);
        acc[nb][c][3] = mfma_16x16x4(T.v[rho][c].w, pr[rho], acc[nb][c][3]);
      }
  }
}

// ---------------------------------------------------------------------------
// Static part of the schedule.
//
// Rows are scheduled in units of Cd rows (one turn of the tile ring for all
// four waves).  Every slab of sequence b holds st(b) = floor(fnum/16 * n_b /
// Cd) static units at its start (ceil(n_b / Cd), all of it, for fnum = 16);
// the rest of its rows is its dynamic part,
// handed out one unit at a time.  The static units of all slabs, in slab
// order, form one space of Ru units that is cut into gridDim.x contiguous
// ranges, [w*Ru/G, (w+1)*Ru/G) for workgroup w: the ranges are proportional
// to the rows, so every workgroup starts with the same amount of work (to
// one unit) and without touching a counter.  A range covers one or more
// slabs; each (workgroup, slab) pair is a visit with its own partial slot.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int static_units(int n_b, int Cd, int fnum) {
  if (fnum >= kStaticDen) return (n_b + Cd - 1) / Cd;          // the whole slab
  return (int)((int64_t)n_b * fnum / ((int64_t)kStaticDen * Cd));
}

// Units of the dynamic part of a slab with n rows.
__device__ __forceinline__ int dynamic_units(int n, int Cd, int fnum) {
  const int rest = n - static_units(n, Cd, fnum) * Cd;
  return rest > 0 ? (rest + Cd - 1) / Cd : 0;
}

__device__ __forceinline__ int64_t wave_incl_scan(int64_t v, int lane) {
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int64_t o = __shfl_up(v, d);
    if (lane >= d) v += o;
  }
  return v;
}

// Wave-wide (all 64 lanes).  Static units of one slab of sequence `bq` and
// of one slab of each sequence before it; returns the static units of one
// slab summed over all sequences.
__device__ int64_t static_scan(const int32_t* __restrict__ len, int B, int n_max, bool app, int T,
                               int Cd, int fnum, int bq, int lane, int64_t* before, int* st_bq) {
  int64_t carry = 0;
  for (int b0 = 0; b0 < B; b0 += kWave) {
    const int b = b0 + lane;
    const int64_t v = b < B ? static_units(decode_rows(len[b], n_max, app, T), Cd, fnum) : 0;
    const int64_t incl = wave_incl_scan(v, lane);
    if (bq >= b0 && bq < b0 + kWave) {
      *before = carry + __shfl(incl - v, bq - b0);
      *st_bq = (int)__shfl(v, bq - b0);
    }
    carry += __shfl(incl, kWave - 1);
  }
  return carry;
}

// Wave-wide.  The sequence whose slabs hold static unit u (a sequence holds
// per_b times the static units of one of its slabs); *first = its first
// unit, *st = its static units per slab.  -1 if u lies beyond every static
// unit.
__device__ int static_locate(const int32_t* __restrict__ len, int B, int n_max, bool app, int T,
                             int Cd, int fnum, int per_b, int64_t u, int lane, int64_t* first,
                             int* st) {
  int64_t carry = 0;
  for (int b0 = 0; b0 < B; b0 += kWave) {
    const int b = b0 + lane;
    const int64_t v =
        b < B ? (int64_t)per_b * static_units(decode_rows(len[b], n_max, app, T), Cd, fnum) : 0;
    const int64_t incl = wave_incl_scan(v, lane);
    const unsigned long long m = __ballot(carry + incl > u);
    if (m) {
      const int f = __ffsll((long long)m) - 1;
      *first = carry + __shfl(incl - v, f);
      *st = (int)(__shfl(v, f) / per_b);
      return b0 + f;
    }
    carry += __shfl(incl, kWave - 1);
  }
  return -1;
}

__device__ __forceinline__ int64_t ceil_div64(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Static visits (= partial slots) of a slab whose static units are units
// [Ps, Ps + st) of Ru, cut G ways.  With Ru >= G every workgroup whose range
// meets the slab has a slot, numbered from the first such workgroup; with
// Ru < G every range is at most one unit and the slot is the unit's index in
// the slab (workgroups with an empty range take none).
__device__ __forceinline__ int static_visits(int64_t Ps, int st, int64_t Ru, int G) {
  if (st <= 0) return 0;
  if (Ru < G) return st;
  const int64_t wf = ceil_div64((Ps + 1) * G, Ru) - 1;
  const int64_t wl = ceil_div64((Ps + st) * G, Ru) - 1;
  return (int)(wl - wf + 1);
}

__device__ __forceinline__ int static_slot(int64_t Ps, int64_t u, int64_t Ru, int G, int w) {
  if (Ru < G) return (int)(u - Ps);
  return (int)(w - (ceil_div64((Ps + 1) * G, Ru) - 1));
}

// Number of cache rows of slab s = (b, KV head, head group).
__device__ __forceinline__ int slab_rows(const int32_t* __restrict__ len, int s, int per_b,
                                         int n_max, bool app, int T) {
  return decode_rows(len[s / per_b], n_max, app, T);
}

__device__ __forceinline__ unsigned long long load_word(const unsigned long long* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Wave-wide search (all 64 lanes call it): the first slab at or after
// `start` (cyclically) that still has dynamic units and visit slots left, looking
// at no more than `budget` slabs.  Returns -1 if none; *seen is the number of
// slabs examined up to and including the one returned.
__device__ int find_open_slab(const unsigned* __restrict__ cnt,
                              const int32_t* __restrict__ len, int start, int budget, int S,
                              int per_b, int n_max, bool app, int T, int Cd, int fnum,
                              int J, int lane, int* seen) {
  for (int base = 0; base < budget; base += kWave) {
    const int o = base + lane;
    int sl = start + o;
    if (sl >= S) sl -= S;
    bool open = false;
    if (o < budget) {
      const int nch = dynamic_units(slab_rows(len, sl, per_b, n_max, app, T), Cd, fnum);
      const unsigned long long w = load_word(
          reinterpret_cast<const unsigned long long*>(cnt + (size_t)sl * kCounterStride));
      open = (unsigned)w < (unsigned)nch && (unsigned)(w >> 32) < (unsigned)J;
    }
    const unsigned long long m = __ballot(open);
    if (m) {
      const int first = __ffsll((long long)m) - 1;
      *seen = base + first + 1;
      const int r = start + base + first;
      return r >= S ? r - S : r;
    }
  }
  *seen = budget;
  return -1;
}

// ---------------------------------------------------------------------------
// Partials, persistent form.
//
// A slab is the cache rows of one (b, KV head, head group).  A fixed set of
// workgroups (one per CU and wave slot) stays resident.  Each first works
// through its static range (see "Static part of the schedule" above): one
// "visit" per slab the range meets.  Its last static visit (the home visit)
// then goes on with the dynamic units of the same slab, taken one at a time
// from the slab's counter.  When those run out the workgroup opens dynamic
// visits on other slabs with units left, taking in one atomic step a slot
// after the slab's static ones and the first two units, so every dynamic
// visit has rows and the slots in use are exactly 0 .. visits-1.  A visit
// folds all its rows -- its four waves interleave each segment's 16-row
// tiles, so the workgroup streams one contiguous run of K and of V -- into
// one running (reference, sum, weighted sum) state, since the online softmax does
// not care which rows it has seen, then writes one partial per query head to
// its slot and counts the visit in each head's visit count.  Faster CUs
// simply take more units at the end.  Nothing here waits on another
// workgroup or needs a device-wide fence: the merge, a separate launch, sees
// every partial.
//
//   slab line  per slab one 128-byte line: a 64-bit word {dynamic units
//              taken (low), dynamic visits opened (high)}; reset by the merge
//   nvis       [B][h_q] uint32 visits per query head; reset by the merge
//   ws_ml      [B][h_q][J] float2        (reference, base-2 units; sum)
//   ws_acc     [B][h_q][J][DV]           unnormalised weighted sum of V rows
// ---------------------------------------------------------------------------
template <int DK, int DV, int NB, bool CAUSAL, int W>
__global__ __launch_bounds__(kThreads, W) void decode_partial_kernel(
    const float* __restrict__ q, float* __restrict__ K,
    float* __restrict__ V, const float* __restrict__ k_new,
    const float* __restrict__ v_new, const int32_t* __restrict__ len, float qscale,
    int B, int h_q, int h_kv, int n_max, int T, int C, int Cd, int fnum, int head_groups, int J,
    int Jd, unsigned* __restrict__ cnt, unsigned* __restrict__ nvis, float2* __restrict__ ws_ml,
    float* __restrict__ ws_acc, float* __restrict__ out_direct, int32_t* len_bump) {
  // Two waves per SIMD serve the direct form (out_direct set; nothing is
  // scheduled) and whole-slab static ranges (fnum = 16): nothing is claimed
  // or searched for, so that code compiles away there.
  constexpr bool kTwo = W == 2;
  const int per_b = h_kv * head_groups;
  const int S = B * per_b;
  const int G = h_q / h_kv;
  const bool app = k_new != nullptr;                    // fused append (eqs. (6)-(7))

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);   // wave-uniform
  const int i = lane & 15;
  const int k = lane >> 4;

  __shared__ int sh_ctl[7];      // slab, slot, static rows [sr, er), units d0 d1, dynamic
  __shared__ int sh_next[2];     // dynamic unit after next, by parity
  __shared__ f4 sh_q[NB][DK / 16][kWave];
  __shared__ f4 sh_acc[kWaves - 1][NB][DV / 64][4][kWave];
  __shared__ float sh_m[kWaves - 1][NB][kWave];
  __shared__ float sh_l[kWaves - 1][NB][kWave];
  // Row-pair layout: each wave's K tile, 16 slots of d_k + 4 floats.
  constexpr bool PAIRS = kPairs<NB, W>;
  __shared__ __align__(16) char sh_k[PAIRS ? kWaves : 1][PAIRS ? 16 * kKSlot<DK> : 16];

  // Fused append: rows len[b] + r of KV head u = (b, g) <- k_new / v_new row
  // r (those that fit), bit for bit.  The decode never reads those rows from
  // the cache (it takes them straight from k_new / v_new), so no ordering
  // between the copies and the reads is needed.  len[b] is advanced only
  // once every workgroup has read it: by the merge, or in the direct form by
  // the sequence's last workgroup (see the end of this kernel).
  constexpr int ck = DK / 4, cv = DV / 4;               // 16-byte chunks per row
  auto append_rows = [&](int u, int32_t t) {
    const int cnt = appended_rows(app, t, n_max, T);
    for (int w = tid; w < cnt * (ck + cv); w += kThreads) {
      const int r = w / (ck + cv);
      const int x = w - r * (ck + cv);
      const int64_t row = (int64_t)u * n_max + t + r;
      const int64_t src = (int64_t)u * T + r;
      if (x < ck)
        reinterpret_cast<u4*>(K + row * DK)[x] = reinterpret_cast<const u4*>(k_new + src * DK)[x];
      else
        reinterpret_cast<u4*>(V + row * DV)[x - ck] =
            reinterpret_cast<const u4*>(v_new + src * DV)[x - ck];
    }
  };
  // Persistent form: the workgroups share the copies up front.
  if (!out_direct && app)
    for (int u = blockIdx.x; u < B * h_kv; u += gridDim.x) append_rows(u, len[u / h_kv]);
  int start = (int)(((int64_t)blockIdx.x * S) / gridDim.x);
  // Direct form (out_direct set; every slab is a single chunk): workgroup s
  // owns slab s, takes its one chunk without searching and writes the output
  // rows itself -- no merge, and no other workgroup touches its counter line.
  bool first = true;
  // This workgroup's static range, units [u_lo, u_hi) of Ru (wave 0 only).
  const int Gw = (int)gridDim.x;
  const int rank = (int)blockIdx.x;
  int64_t Ru = 0, u_lo = 0, u_hi = 0;
  int ws_s = -1, ws_st = 0;         // slab and units per slab of the last static visit
  if (wave == 0 && fnum > 0) {
    int64_t before;
    int st;
    Ru = (int64_t)per_b * static_scan(len, B, n_max, app, T, Cd, fnum, -1, lane, &before, &st);
    u_lo = (int64_t)rank * Ru / Gw;
    u_hi = (int64_t)(rank + 1) * Ru / Gw;
  }

  while (true) {
    // ---- wave 0 opens a visit.  First the static visits of this
    // workgroup's range, one per slab the range meets; the last of them (the
    // home visit) goes on with the dynamic units of its slab.  Then dynamic
    // visits on any slab with dynamic units and slots left: lane 0 takes the
    // slot and the first two units with one compare-and-swap on the slab's
    // {units, visits} word, so every such visit has at least one unit and
    // no slab gets more than Jd of them.
    if (wave == 0) {
      int s = -1, j = -1, sr = 0, er = 0, d0 = -1, d1 = -1, dyn = 0;
      int budget = (kTwo || out_direct || fnum >= kStaticDen) ? 0 : S;
      if (out_direct) {
        if (first) {
          s = blockIdx.x;
          j = 0;
          er = C;
        }
      } else if (u_lo < u_hi) {
        // The slab holding unit u_lo.  A static visit that is not the last
        // of its range ends at its slab's end, so with whole-slab ranges the
        // next visit is the next slab of the same sequence (same units) if
        // there is one; otherwise a search over the sequences' prefix sums.
        int64_t fu = 0;
        int stb = 0, bs, r;
        int64_t Ps;
        if (fnum >= kStaticDen && ws_s >= 0 && (ws_s + 1) % per_b != 0) {
          bs = (ws_s + 1) / per_b;
          r = (ws_s + 1) % per_b;
          stb = ws_st;
          Ps = u_lo;
        } else {
          bs = static_locate(len, B, n_max, app, T, Cd, fnum, per_b, u_lo, lane, &fu, &stb);
          r = stb > 0 ? (int)((u_lo - fu) / stb) : 0;
          Ps = fu + (int64_t)r * stb;
        }
        if (bs >= 0 && stb > 0) {
          const int64_t e = u_hi < Ps + stb ? u_hi : Ps + stb;
          s = bs * per_b + r;
          j = static_slot(Ps, u_lo, Ru, Gw, rank);
          sr = (int)(u_lo - Ps) * Cd;
          er = (int)(e - Ps) * Cd;
          u_lo = e;
          ws_s = s;
          ws_st = stb;
          budget = 0;
          if (!kTwo && u_lo == u_hi && fnum < kStaticDen) {
            // The home visit.  If its static rows do not fill the
            // two-segment window, its first dynamic units are taken now.
            dyn = 1;
            start = s;
            const int nseg = (er - sr + C - 1) / C;
            if (nseg < 2) {
              unsigned long long got = 0;
              if (lane == 0)
                got = atomicAdd(
                    reinterpret_cast<unsigned long long*>(cnt + (size_t)s * kCounterStride),
                    (unsigned long long)(2 - nseg));
              got = __shfl(got, 0);
              d0 = (int)(unsigned)got;
              d1 = d0 + 1;
            }
          }
        } else {
          u_lo = u_hi;
        }
      }
      while (!kTwo && budget > 0) {
        int seen;
        const int cand = find_open_slab(cnt, len, start, budget, S, per_b, n_max, app, T, Cd,
                                        fnum, Jd, lane, &seen);
        if (cand < 0) break;
        budget -= seen;
        start = cand + 1 == S ? 0 : cand + 1;
        const int nch = dynamic_units(slab_rows(len, cand, per_b, n_max, app, T), Cd, fnum);
        unsigned long long got = ~0ull;
        if (lane == 0) {
          unsigned long long* w =
              reinterpret_cast<unsigned long long*>(cnt + (size_t)cand * kCounterStride);
          unsigned long long old = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          // Lock-free: a failed swap means another workgroup moved the word.
          while ((unsigned)old < (unsigned)nch && (unsigned)(old >> 32) < (unsigned)Jd) {
            const unsigned long long seen_w = atomicCAS(w, old, old + (1ull << 32) + 2ull);
            if (seen_w == old) {
              got = old;
              break;
            }
            old = seen_w;
          }
        }
        got = __shfl(got, 0);
        if (got == ~0ull) continue;                     // no unit or slot left meanwhile
        s = cand;
        d0 = (int)(unsigned)got;
        d1 = d0 + 1;
        dyn = 1;
        // Dynamic slots follow the slab's static ones.
        int base = 0;
        if (fnum > 0) {
          int64_t before = 0;
          int st = 0;
          static_scan(len, B, n_max, app, T, Cd, fnum, cand / per_b, lane, &before, &st);
          base = static_visits((int64_t)per_b * before + (int64_t)(cand % per_b) * st, st, Ru, Gw);
        }
        j = base + (int)(got >> 32);
        break;
      }
      if (lane == 0) {
        sh_ctl[0] = s;
        sh_ctl[1] = j;
        sh_ctl[2] = sr;
        sh_ctl[3] = er;
        sh_ctl[4] = d0;
        sh_ctl[5] = d1;
        sh_ctl[6] = dyn;
      }
    }
    __syncthreads();
    const int s = sh_ctl[0];
    const int j = sh_ctl[1];
    const int sr = sh_ctl[2];
    const int er = sh_ctl[3];
    const int d0 = sh_ctl[4];
    const int d1 = sh_ctl[5];
    const bool dyn = !kTwo && sh_ctl[6] != 0;
    if (s < 0) break;                                   // every slab is exhausted
    first = false;

    const int b = s / per_b;
    const int rem = s - b * per_b;
    const int g = rem / head_groups;
    const int hgrp = rem - g * head_groups;
    const int32_t len_b = len[b];
    const int n = decode_rows(len_b, n_max, app, T);
    const int last_row = n - 1;
    if (out_direct && n == 0) {
      // An empty cache: the slab's output rows are zero.
      const int hc = min(NB * kHeadsPerBlock, G - hgrp * (NB * kHeadsPerBlock));
      float* o = out_direct + ((int64_t)b * h_q + g * G + hgrp * (NB * kHeadsPerBlock)) * DV;
      for (int e = tid; e < hc * (DV / 4); e += kThreads)
        reinterpret_cast<f4*>(o)[e] = f4{0.f, 0.f, 0.f, 0.f};
      break;
    }
    const int h_first = g * G + hgrp * (NB * kHeadsPerBlock);
    const int h_count = min(NB * kHeadsPerBlock, G - hgrp * (NB * kHeadsPerBlock));
    const int64_t slab = (int64_t)b * h_kv + g;
    unsigned long long* slab_word =
        reinterpret_cast<unsigned long long*>(cnt + (size_t)s * kCounterStride);
    RowSource src;
    src.Ks = K + slab * n_max * DK;
    src.Vs = V + slab * n_max * DV;
    src.new_cnt = appended_rows(app, len_b, n_max, T);
    src.new_lo = src.new_cnt > 0 ? len_b : n;
    src.new_row = src.new_cnt == 1 ? len_b : -1;
    src.fast_end = src.new_lo;
    src.k_new_rows = app ? k_new + slab * T * DK : nullptr;
    src.v_new_rows = app ? v_new + slab * T * DV : nullptr;
    src.k_lane = (uint32_t)(i * DK + 4 * k) * sizeof(float);
    src.v_lane = (uint32_t)(4 * k * DV + 4 * i) * sizeof(float);
    src.first_off = kTileRows * wave;
    if constexpr (PAIRS) pair_lane_setup<DK, DV>(src, wave, i, k);

    // Last row each lane's column sees.  A causal column is query row
    // r = (its index in the KV head's group) mod T, at position pos0 + r:
    // pos0 = len[b] before a fused append (the rows of one step enter one per
    // position), else n - T (the last T positions of the cache).
    int lim[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      lim[nb] = last_row;
      if constexpr (CAUSAL) {
        const int vh = hgrp * (NB * kHeadsPerBlock) + nb * kHeadsPerBlock + i;
        const int pos0 = app ? (int)len_b : n - T;
        lim[nb] = (int)std::min<int64_t>((int64_t)pos0 + vh % T, last_row);
      }
    }

    // The visit's rows are a stream of segments: its static rows [sr, er)
    // in segments of up to C rows, then, for the home visit and dynamic
    // visits, the slab's dynamic units in the order its counter hands them
    // out (Cd rows each, from row srows on).  The workgroup always knows the
    // current segment (start row cs, ctpw tiles per wave) and the next one
    // (ns < 0: none); a dynamic segment after next is requested at the start
    // of each segment.  A wave's tiles of a segment start at rows cs + x*64 +
    // wave*16, x < ctpw.  The register tiles form a ring: while one tile is
    // on the matrix cores the loads of the next R-1 are in flight, across
    // segment boundaries too (past the visit's end the clamped last row,
    // already cached, is loaded so every path keeps the same loads in flight).
    constexpr int kRowsPerTurn = kWaves * kTileRows;
    const int srows = static_units(n, Cd, fnum) * Cd;
    const int nchd = dynamic_units(n, Cd, fnum);
    const int tpw_d = Cd / kRowsPerTurn;
    auto dyn_row = [&](int d) { return d >= 0 && d < nchd ? srows + d * Cd : -1; };
    auto static_tpw = [&](int at) { return min(C, er - at) / kRowsPerTurn; };
    int snext = sr;                                     // next static segment not yet entered
    int cs, ctpw, ns, ntpw;
    bool d0_used = false;
    if (snext < er) {
      cs = snext;
      ctpw = static_tpw(snext);
      snext += C;
    } else {
      cs = dyn ? dyn_row(d0) : -1;
      ctpw = tpw_d;
      d0_used = true;
    }
    if (snext < er) {
      ns = snext;
      ntpw = static_tpw(snext);
      snext += C;
    } else {
      ns = dyn ? dyn_row(d0_used ? d1 : d0) : -1;
      ntpw = tpw_d;
    }
    // First row of the wave's tile x of the stream (its smallest row).
    auto row_of = [&](int x) {
      return x < ctpw ? cs + x * kRowsPerTurn + src.first_off
                      : (ns >= 0 ? ns + (x - ctpw) * kRowsPerTurn + src.first_off : last_row);
    };
    // B operand of the score product: lane (k, i) holds q of head nb*16+i at
    // dims 16t+4k..+3, scaled into base-2 units (zero for the padding heads
    // of a partial column block).  Where it is held in registers for the
    // whole visit, every wave loads it straight into that layout; otherwise
    // it is staged once in LDS in register order and re-read for every tile.
    // Either way the q loads go out first and the ring's first tiles right
    // after them, so the wait for q leaves the tiles in flight.
    constexpr bool kPin = W == 1 && kPinQ<NB, DK>;
    constexpr int kQPerThread = NB * (DK / 16) * kWave / kThreads;
    static_assert(kQPerThread * kThreads == NB * (DK / 16) * kWave, "q staging");
    f4 qr[NB][DK / 16];
    f4 qv[kPin ? 1 : kQPerThread];
    if constexpr (kPin) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int hl = nb * kHeadsPerBlock + i;
        const float* qh = q + ((int64_t)b * h_q + h_first + hl) * DK + 4 * k;
#pragma unroll
        for (int t = 0; t < DK / 16; ++t)
          qr[nb][t] = hl < h_count ? load4(qh + 16 * t) : f4{0.f, 0.f, 0.f, 0.f};
      }
    } else {
#pragma unroll
      for (int u = 0; u < kQPerThread; ++u) {
        const int e = tid + u * kThreads;
        const int ln = e % kWave;
        const int t = (e / kWave) % (DK / 16);
        const int nb = e / (kWave * (DK / 16));
        const int hl = nb * kHeadsPerBlock + (ln & 15);
        qv[u] = f4{0.f, 0.f, 0.f, 0.f};
        if (hl < h_count)
          qv[u] = load4(q + ((int64_t)b * h_q + h_first + hl) * DK + 16 * t + 4 * (ln >> 4));
      }
    }
    constexpr int R = W == 2 ? 2 : kRing<NB, DK, DV>;
    Tile<DK, DV, NB> ring[R];
    auto load = [&](Tile<DK, DV, NB>& T, int row0, int lr) {
      if constexpr (PAIRS) load_tile_pairs<DK, DV, NB, CAUSAL>(T, src, row0, lr, lane);
      else load_tile<DK, DV, NB, CAUSAL>(T, src, row0, lr, i, k);
    };
    // (Unconditional, so that the wait for q counts only the q loads; a
    // visit without rows, which the schedule never opens, would read row 0.)
#pragma unroll
    for (int p = 0; p < R - 1; ++p)
      load(ring[p], cs >= 0 ? row_of(p) : 0, max(last_row, 0));
    if constexpr (kPin) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int t = 0; t < DK / 16; ++t) qr[nb][t] *= qscale;
    } else {
#pragma unroll
      for (int u = 0; u < kQPerThread; ++u) {
        const int e = tid + u * kThreads;
        sh_q[e / (kWave * (DK / 16))][(e / kWave) % (DK / 16)][e % kWave] = qv[u] * qscale;
      }
      __syncthreads();
    }

    // Running state per column block; lane (k, i) belongs to head i.
    float m_run[NB], l_run[NB];
    f4 acc[NB][DV / 64][4];   // acc[nb][c][e][r] = O[dim 64c+16k+4r+e][head i]
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      m_run[nb] = -INFINITY;
      l_run[nb] = 0.f;
#pragma unroll
      for (int cc = 0; cc < DV / 64; ++cc)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[nb][cc][e] = f4{0.f, 0.f, 0.f, 0.f};
    }

    if (cs >= 0) {
      for (int it = 0;; ++it) {
        // The segment after next comes from the counter once the static
        // rows are all in the window.  Its value is left undefined for the
        // threads that do not ask (rather than merged with a default): a
        // merge right here would make the compiler wait for the request, and
        // with it for every prefetched tile load.
        const bool req = dyn && ns >= 0 && snext >= er;
        int after;
        if (tid == 0 && req) after = (int)(unsigned)atomicAdd(slab_word, 1ull);
        // A loop that always runs at least once and exits at its bottom:
        // after its first wait on a tile load the compiler knows the request
        // issued above (an older memory operation) has returned, so
        // publishing its value below costs no wait that would drain the
        // prefetched tiles.  Each turn of the ring loads tile t+p+R-1 into
        // the slot tile t+p-1 has just left, then processes tile t+p (all
        // indices are constants after unrolling, so the ring lives in
        // registers).
        int t = 0;
        do {
#pragma unroll
          for (int p = 0; p < R; ++p) {
            const int r = row_of(t + p);
            load(ring[(p + R - 1) % R], row_of(t + p + R - 1), last_row);
            if (r <= last_row) {
              if constexpr (PAIRS)
                process_tile_pairs<DK, DV, NB, CAUSAL, kPin>(ring[p], r, lim, src, lane,
                                                             sh_k[PAIRS ? wave : 0], sh_q, qr,
                                                             m_run, l_run, acc);
              else
                process_tile<DK, DV, NB, CAUSAL, kPin>(ring[p], r, lim, k, lane, sh_q, qr, m_run,
                                                       l_run, acc);
            }
          }
          t += R;
          // A wave whose remaining tiles all lie past the slab's end (only
          // in the slab's last segment) leaves early instead of idling through
          // them.
        } while (t < ctpw && row_of(t) <= last_row);
        // Only a segment that requested a unit publishes it (and such
        // segments are consecutive: the dynamic tail of the visit); the static
        // segments before it need no barrier -- every wave derives the same
        // segment stream by itself.
        if (req) {
          if (tid == 0) sh_next[it & 1] = after;
          __syncthreads();
        }
        cs = ns;
        ctpw = ntpw;
        if (cs < 0) break;
        if (snext < er) {
          ns = snext;
          ntpw = static_tpw(snext);
          snext += C;
        } else {
          ns = req ? dyn_row(sh_next[it & 1]) : -1;
          ntpw = tpw_d;
        }
      }
    }

    // Row sums of head i are spread over the 4 row groups k.
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      l_run[nb] = sum_over_row_groups(l_run[nb]);
    }

    // Combine the 4 waves: waves 1..3 park their state in LDS in their own
    // register layout; wave 0 rescales and adds it lane by lane, writes the
    // visit's partial and counts the visit for each of its heads.
    if (wave > 0) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        sh_m[wave - 1][nb][lane] = m_run[nb];
        sh_l[wave - 1][nb][lane] = l_run[nb];
#pragma unroll
        for (int cc = 0; cc < DV / 64; ++cc)
#pragma unroll
          for (int e = 0; e < 4; ++e) sh_acc[wave - 1][nb][cc][e][lane] = acc[nb][cc][e];
      }
    }
    __syncthreads();
    if (wave == 0) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        // Wave 0 always holds the visit's first row, so M is finite (unless
        // a causal column sees none of the visit's rows); a wave that saw no
        // row has m = -inf and weight exp2(-inf) = 0.
        float M = m_run[nb];
#pragma unroll
        for (int w = 0; w < kWaves - 1; ++w) M = fmaxf(M, sh_m[w][nb][lane]);
        float M_ref = M;
        if constexpr (CAUSAL) M_ref = M == -INFINITY ? 0.f : M;
        const float w0 = fast_exp2(m_run[nb] - M_ref);
        float L = l_run[nb] * w0;
#pragma unroll
        for (int cc = 0; cc < DV / 64; ++cc)
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[nb][cc][e] *= w0;
#pragma unroll
        for (int w = 0; w < kWaves - 1; ++w) {
          const float ww = fast_exp2(sh_m[w][nb][lane] - M_ref);
          L += sh_l[w][nb][lane] * ww;
#pragma unroll
          for (int cc = 0; cc < DV / 64; ++cc)
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[nb][cc][e] += sh_acc[w][nb][cc][e][lane] * ww;
        }
        const int hl = nb * kHeadsPerBlock + i;
        if (hl < h_count) {
          const int64_t head = (int64_t)b * h_q + h_first + hl;
          const int64_t slot = head * J + j;
          float* dst;
          float inv = 1.f;
          if (out_direct) {
            // The only visit of the slab: normalise and write the output row
            // (a causal row that saw no key, L = 0, gives zeros).
            dst = out_direct + head * DV;
            inv = L > 0.f ? 1.f / L : 0.f;
          } else {
            dst = ws_acc + slot * DV;
            if (k == 0) {
              ws_ml[slot] = make_float2(M, L);
              atomicAdd(nvis + head, 1u);
            }
          }
#pragma unroll
          for (int cc = 0; cc < DV / 64; ++cc)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const f4 o = f4{acc[nb][cc][0][r], acc[nb][cc][1][r], acc[nb][cc][2][r],
                              acc[nb][cc][3][r]};
              *reinterpret_cast<f4*>(dst + 64 * cc + 16 * k + 4 * r) = o * inv;
            }
        }
      }
    }
    if (out_direct) {
      // Thread 0 issued this slab's only counter requests; clear the line
      // for the next call (program order keeps the store after them).
      if (tid == 0)
        *reinterpret_cast<unsigned long long*>(cnt + (size_t)s * kCounterStride) = 0ull;
      break;
    }
    // Wave 0 runs the next search; the barrier at its end keeps the other
    // waves from touching sh_q / sh_ctl before wave 0 is done here.
  }

  // Direct form of a fused append (the whole step in this one launch; two
  // waves per SIMD, the only direct form that takes one): the
  // first head group of each KV head copies its rows, then every workgroup
  // of sequence b checks in on the sequence's counter (word 2 of the line of
  // its first slab) once all its waves are done reading len[b].  The last to
  // check in advances len[b] by the rows that fit and clears the counter for
  // the next call.
  if (kTwo && out_direct && app) {
    const int sd = (int)blockIdx.x;
    const int b = sd / per_b;
    const int rem = sd - b * per_b;
    const int g = rem / head_groups;
    const int32_t t = len[b];
    if (rem - g * head_groups == 0) append_rows(b * h_kv + g, t);
    // Every wave has read len[b] (its copies depend on it) before the check-in.
    __syncthreads();
    if (tid == 0 && len_bump) {
      unsigned* arrivals = cnt + (size_t)b * per_b * kCounterStride + 2;
      if (atomicAdd(arrivals, 1u) == (unsigned)per_b - 1u) {
        *arrivals = 0u;
        if (t >= 0 && t < n_max) len_bump[b] = t + min(T, n_max - t);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Merge, one workgroup per (slab, query head of its group): eqs. (2)-(3)
// regrouped over disjoint row sets,
//   out[b,h,:] = sum_j 2^(m_j - M) acc_j / sum_j 2^(m_j - M) l_j,  M = max_j m_j,
// over the head's nv visit partials (nv = 0: an empty cache, out = 0).
// Threads split the visits kLanesV ways and the 16-byte columns DV/4 ways,
// then combine through LDS.  Every piece of scheduling state is reset by the
// one workgroup that owns it -- the head's visit count by its workgroup, the
// slab's line by the slab's first head -- so the next call finds zeros, with
// no atomics and no device-wide fences.
// ---------------------------------------------------------------------------
template <int DV>
__global__ __launch_bounds__(kThreads) void decode_merge_kernel(
    float* __restrict__ out, const float2* __restrict__ ws_ml,
    const float* __restrict__ ws_acc, int h_q, int h_kv, int head_groups, int heads_per_group,
    int merge_heads, int J, unsigned* __restrict__ cnt, unsigned* __restrict__ nvis,
    int32_t* __restrict__ len_bump, int n_max, int T) {
  constexpr int kCols = DV / 4;                         // 16-byte columns per row
  constexpr int kLanesV = kThreads / kCols;             // visits merged in parallel
  const int s = blockIdx.x / merge_heads;
  const int hl = blockIdx.x - s * merge_heads;
  const int per_b = h_kv * head_groups;
  const int b = s / per_b;
  const int rem = s - b * per_b;
  const int g = rem / head_groups;
  const int hgrp = rem - g * head_groups;
  const int G = h_q / h_kv;
  const int h_count = min(heads_per_group, G - hgrp * heads_per_group);
  if (hl >= h_count) return;                            // padding workgroup
  const int tid = threadIdx.x;
  const int64_t row = (int64_t)b * h_q + g * G + hgrp * heads_per_group + hl;
  const int ch = tid % kCols;
  const int pv = tid / kCols;
  const float2* ml = ws_ml + row * J;
  const float* acc = ws_acc + row * J * DV;
  // This lane's first visit (slot pv) is loaded together with the visit
  // count, before it is known whether the slot holds a visit (it is used
  // only if it does), so that a head with at most kLanesV visits takes one
  // round trip to memory.
  float2 st0 = make_float2(-INFINITY, 0.f);
  f4 a0 = f4{0.f, 0.f, 0.f, 0.f};
  if (pv < J) {
    st0 = ml[pv];
    a0 = load4(acc + (int64_t)pv * DV + 4 * ch);
  }
  const int nv = min((int)nvis[row], J);

  // This lane's visits pv, pv + kLanesV, ...: a running reference (the
  // largest so far), sum and weighted sum, rescaled when the reference
  // rises; a visit that saw no row (reference -inf) adds nothing.
  float m = -INFINITY, l = 0.f;
  f4 o = f4{0.f, 0.f, 0.f, 0.f};
  auto add = [&](float2 st, f4 a) {
    if (st.x == -INFINITY) return;
    const float mn = fmaxf(m, st.x);
    const float wo = fast_exp2(m - mn);                 // 0 while m = -inf
    const float wn = fast_exp2(st.x - mn);
    l = l * wo + st.y * wn;
    o = o * wo + a * wn;
    m = mn;
  };
  if (pv < nv) add(st0, a0);
  for (int jj = pv + kLanesV; jj < nv; jj += kLanesV)
    add(ml[jj], load4(acc + (int64_t)jj * DV + 4 * ch));
  __shared__ float sh_m[kThreads], sh_l[kThreads];
  __shared__ f4 sh_o[kThreads];
  sh_m[tid] = m;
  sh_l[tid] = l;
  sh_o[tid] = o;
  __syncthreads();
  if (pv == 0) {
    float M = m;
    for (int p = 1; p < kLanesV; ++p) M = fmaxf(M, sh_m[p * kCols + ch]);
    float L = 0.f;
    f4 O = f4{0.f, 0.f, 0.f, 0.f};
    if (M != -INFINITY) {
      for (int p = 0; p < kLanesV; ++p) {
        const float w = fast_exp2(sh_m[p * kCols + ch] - M);
        L += sh_l[p * kCols + ch] * w;
        O += sh_o[p * kCols + ch] * w;
      }
    }
    *reinterpret_cast<f4*>(out + row * DV + 4 * ch) =
        M != -INFINITY ? O / L : f4{0.f, 0.f, 0.f, 0.f};
  }
  if (tid == 0) {
    nvis[row] = 0u;
    if (hl == 0) {
      // The slab's line: read by no merge workgroup, so its first head's
      // workgroup clears it.
      *reinterpret_cast<unsigned long long*>(cnt + (size_t)s * kCounterStride) = 0ull;
      // Completing a fused append: len[b] advances once per sequence (by
      // the rows that fit), after the partial kernel (which read it) has
      // finished.
      if (len_bump && g == 0 && hgrp == 0) {
        const int32_t t = len_bump[b];
        if (t >= 0 && t < n_max) len_bump[b] = t + min(T, n_max - t);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Host side: validation, sizing, launches.
// ---------------------------------------------------------------------------
struct Plan {
  int chunk_rows;     // most rows per segment
  int dyn_rows;       // rows per scheduling unit (one ring turn of the 4 waves)
  int fnum;           // static share of the rows, in sixteenths (0: all dynamic)
  int head_groups;    // groups of up to 32 query heads per KV head
  int blocks;         // MFMA column blocks per wave (1 or 2)
  int slabs;          // B * h_kv * head_groups
  int grid;           // resident workgroups of the partial kernel
  int J;              // visit slots per (b, query head): static, then dynamic
  int Jd;             // dynamic visit slots per slab
  int merge_heads;    // query heads per slab the merge covers
  bool single_chunk;  // every slab fits in one chunk (direct form possible)
  bool two_waves;     // whole-slab static ranges at two workgroups per CU
  size_t line_bytes, counter_bytes, ml_bytes, bytes;
};

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
bool dim_ok(int d) { return d == 64 || d == 128 || d == 256; }
int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
size_t pad256(size_t x) { return (x + 255) / 256 * 256; }

da_status check_shapes(int B, int h_q, int h_kv, int n_max, int d_k, int d_v) {
  if (B < 1 || h_q < 1 || h_kv < 1 || n_max < 1 || d_k < 1 || d_v < 1) return DA_ERR_SHAPE;
  if (h_q % h_kv != 0) return DA_ERR_SHAPE;
  const int64_t slabs = (int64_t)B * h_kv * ceil_div(h_q / h_kv, kHeadsPerGroup);
  if (slabs > kMaxSlabs || (int64_t)B * h_q > kMaxSlabs * kHeadsPerGroup) return DA_ERR_SHAPE;
  if (!dim_ok(d_k) || !dim_ok(d_v)) return DA_ERR_UNSUPPORTED;
  return DA_OK;
}

// Resident workgroups on the current device: its compute units, at most
// kMaxResident, queried once per device.  Without a device (the call can then
// only fail at launch) the bound itself.
constexpr int kMaxDevices = 64;
std::atomic<int> g_device_cus[kMaxDevices];

int device_resident() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return kMaxResident;
  }
  int c = g_device_cus[dev].load(std::memory_order_relaxed);
  if (c == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n < 1) {
      (void)hipGetLastError();
      return kMaxResident;
    }
    c = std::min(n, kMaxResident);
    g_device_cus[dev].store(c, std::memory_order_relaxed);
  }
  return c;
}

// kDynamicMinUnits, or the environment's override (read at every call).
int dynamic_min_units() {
  const char* e = std::getenv("DECODE_ATTN_DYNAMIC_MIN_UNITS");
  if (!e || !*e) return kDynamicMinUnits;
  char* end = nullptr;
  const long v = std::strtol(e, &end, 10);
  return (*end == 0 && v >= 0 && v <= (1L << 20)) ? (int)v : kDynamicMinUnits;
}

// The work decomposition for these shapes with `resident` resident
// workgroups.  Every size below grows with `resident`, so the plan for
// kMaxResident bounds the workspace of any device's plan.
da_status make_plan(int B, int h_q, int h_kv, int n_max, int d_k, int d_v, int chunk_rows,
                    int resident, Plan* plan) {
  da_status st = check_shapes(B, h_q, h_kv, n_max, d_k, d_v);
  if (st != DA_OK) return st;
  const int G = h_q / h_kv;
  if (chunk_rows == 0) {
    // The default, or the whole cache rounded up to the quantum if shorter
    // or if there are many short slabs (see kDirectMinSlabs).
    const int64_t whole = ceil_div(n_max, kChunkQuantum) * kChunkQuantum;
    const int64_t slabs = (int64_t)B * h_kv * ceil_div(G, kHeadsPerGroup);
    chunk_rows = kDefaultChunkRows;
    if (G <= kHeadsPerBlock && d_k + d_v <= 256 && slabs >= kDirectMinSlabs &&
        n_max <= kDirectMaxRows)
      chunk_rows = (int)whole;
    chunk_rows = (int)std::min<int64_t>(chunk_rows, whole);
  }
  if (chunk_rows < kChunkQuantum || chunk_rows % kChunkQuantum != 0) return DA_ERR_SHAPE;
  plan->chunk_rows = chunk_rows;
  plan->head_groups = (int)ceil_div(G, kHeadsPerGroup);
  plan->blocks = G > kHeadsPerBlock ? 2 : 1;
  plan->slabs = B * h_kv * plan->head_groups;
  plan->merge_heads = std::min(G, plan->blocks * kHeadsPerBlock);
  const int64_t chunks_per_slab = ceil_div(n_max, chunk_rows);
  plan->single_chunk = chunks_per_slab == 1;
  // One resident workgroup per CU, fewer if there are fewer chunks than that.
  plan->grid = (int)std::max<int64_t>(1, std::min<int64_t>(resident, chunks_per_slab * plan->slabs));
  // Static share: off for single-chunk caches (direct form) and for batches
  // whose per-workgroup prefix over sequences would be long.  With two or
  // more slabs per workgroup (one column block) the even split of whole
  // slabs balances the grid by itself and the dynamic searches over many
  // slabs are saved (with two column blocks and many slabs the dynamic
  // remainders measured 0-1.5 % faster); with few units per workgroup the
  // dynamic share cannot move work (kDynamicMinUnits).
  const int64_t units =
      (int64_t)plan->slabs * ceil_div(n_max, ring_tiles(plan->blocks, d_k, d_v) * kWaves * kTileRows);
  const bool few = units < (int64_t)dynamic_min_units() * plan->grid;
  plan->fnum = 0;
  if (!plan->single_chunk && B <= kMaxStaticSeqs)
    plan->fnum = (plan->blocks == 1 && (int64_t)plan->slabs >= 2 * (int64_t)plan->grid) || few
                     ? kStaticDen : kStaticNum;
  // Slabs of at most kDirectMaxRows rows (one column block, d_k + d_v <=
  // 256) run as whole-slab ranges at two workgroups per CU (two waves per
  // SIMD, a two-tile ring): one workgroup's visit starts and ends overlap
  // the other's streaming, and the ranges, proportional to the rows, balance
  // ragged batches.  Measured 2-22 % faster than the one-wave schedule on
  // such caches (the most on small, latency-bound batches); on longer slabs,
  // whose ranges are long enough for the one-wave schedule's deeper ring and
  // dynamic balancing to pay, 1.3-7 % slower.  (Independent of the device's
  // CU count, so that the workspace sized for the largest grid covers every
  // device.)  Longer slabs take the same form when the whole batch is short
  // (kTwoWaveMaxUnits) and the static plan applies.
  const bool tw_base = !plan->single_chunk && B <= kMaxStaticSeqs && plan->blocks == 1 &&
                       d_k + d_v <= 256;
  const bool tw_short_batch = units < (int64_t)kTwoWaveMaxUnits * kMaxResident;
  plan->two_waves = tw_base && (n_max <= kDirectMaxRows || (tw_short_batch && few));
  if (plan->two_waves) {
    plan->grid = (int)std::min<int64_t>(2 * (int64_t)resident, chunks_per_slab * plan->slabs);
    plan->fnum = kStaticDen;
  }
  // Scheduling units (static ranges and dynamic hand-outs) are one ring turn
  // of the four waves when there is a static share, else whole chunks.
  const int ring = plan->two_waves ? 2 : ring_tiles(plan->blocks, d_k, d_v);
  plan->dyn_rows = plan->fnum > 0 ? ring * kWaves * kTileRows : chunk_rows;
  // Static slots: at most one per static unit of a slab plus one, and never
  // more than the workgroups.  Dynamic slots: every dynamic visit holds at
  // least one unit; kVisitSlack times the even share of workgroups per slab
  // leaves room for workgroups that move on from finished slabs.
  const int64_t Js =
      plan->fnum > 0 ? std::min<int64_t>(plan->grid, ceil_div(n_max, plan->dyn_rows)) + 1 : 0;
  const int64_t share = ceil_div((int64_t)plan->grid, plan->slabs);
  plan->Jd = (int)std::max<int64_t>(
      1, std::min(ceil_div(n_max, plan->dyn_rows), kVisitSlack * share));
  int64_t J = Js + plan->Jd;
  if (tw_base && tw_short_batch && !plan->two_waves) {
    // The slots of the two-wave form, which the same shapes take under
    // another DECODE_ATTN_DYNAMIC_MIN_UNITS: the workspace a caller sizes
    // must not depend on the environment.
    const int64_t g2 = std::min<int64_t>(2 * (int64_t)resident, chunks_per_slab * plan->slabs);
    const int64_t r2 = 2 * kWaves * kTileRows;
    const int64_t J2 = std::min<int64_t>(g2, ceil_div(n_max, r2)) + 1 +
                       std::max<int64_t>(1, std::min(ceil_div(n_max, r2),
                                                     kVisitSlack * ceil_div(g2, plan->slabs)));
    J = std::max(J, J2);
  }
  plan->J = (int)J;
  const size_t heads = (size_t)B * h_q;
  const size_t slots = heads * plan->J;
  plan->line_bytes = pad256((size_t)plan->slabs * kCounterStride * sizeof(unsigned));
  plan->counter_bytes = plan->line_bytes + pad256(heads * sizeof(unsigned));
  plan->ml_bytes = pad256(slots * sizeof(float2));
  plan->bytes = plan->counter_bytes + plan->ml_bytes + slots * (size_t)d_v * sizeof(float);
  return DA_OK;
}

struct WsView {
  unsigned* cnt;      // per-slab lines
  unsigned* nvis;     // per-head visit counts
  float2* ml;
  float* acc;
};

WsView view(const Plan& pl, void* workspace) {
  char* base = static_cast<char*>(workspace);
  WsView w;
  w.cnt = reinterpret_cast<unsigned*>(base);
  w.nvis = reinterpret_cast<unsigned*>(base + pl.line_bytes);
  w.ml = reinterpret_cast<float2*>(base + pl.counter_bytes);
  w.acc = reinterpret_cast<float*>(base + pl.counter_bytes + pl.ml_bytes);
  return w;
}

da_status launch_status() {
  return hipGetLastError() == hipSuccess ? DA_OK : DA_ERR_HIP;
}

struct PartialArgs {
  const float* q;
  float* K;
  float* V;
  const float* k_new;   // both NULL: plain decode; both set: fused append
  const float* v_new;
  const int32_t* len;
  float qscale;
  int B, h_q, h_kv, n_max;   // h_q counts query rows: heads x T
  int T;                     // query rows per head (1: single-query decode)
  float* out_direct;         // set: single-chunk slabs, output written directly
  int32_t* len_bump;         // direct form of a fused append: len, advanced in the kernel
};

// The direct form runs two waves per SIMD for one column block and
// d_k + d_v <= 256; only that form takes a fused append.
bool direct_two_waves(const Plan& pl, int d_k, int d_v) {
  return pl.single_chunk && pl.blocks == 1 && d_k + d_v <= 256;
}

template <int DK, int DV, int NB, bool CAUSAL>
void launch_partial(const Plan& pl, const PartialArgs& a, const WsView& w, hipStream_t stream) {
  // The direct form runs one workgroup per slab; otherwise the resident grid.
  const unsigned grid = a.out_direct ? (unsigned)pl.slabs : (unsigned)pl.grid;
  // The direct form schedules nothing: no static share.  The two-wave
  // instances run the direct form of the shapes direct_two_waves() names
  // and the two-wave whole-slab ranges.
  if constexpr (NB == 1 && DK + DV <= 256) {
    if (a.out_direct || pl.two_waves) {
      hipLaunchKernelGGL((decode_partial_kernel<DK, DV, NB, CAUSAL, 2>), dim3(grid),
                         dim3(kThreads), 0, stream, a.q, a.K, a.V, a.k_new, a.v_new, a.len,
                         a.qscale, a.B, a.h_q, a.h_kv, a.n_max, a.T, pl.chunk_rows, pl.dyn_rows,
                         a.out_direct ? 0 : pl.fnum, pl.head_groups, pl.J, pl.Jd, w.cnt, w.nvis,
                         w.ml, w.acc, a.out_direct, a.len_bump);
      return;
    }
  }
  hipLaunchKernelGGL((decode_partial_kernel<DK, DV, NB, CAUSAL, 1>), dim3(grid), dim3(kThreads),
                     0, stream, a.q, a.K, a.V, a.k_new, a.v_new, a.len, a.qscale, a.B, a.h_q,
                     a.h_kv, a.n_max, a.T, pl.chunk_rows, pl.dyn_rows,
                     a.out_direct ? 0 : pl.fnum, pl.head_groups, pl.J, pl.Jd, w.cnt, w.nvis,
                     w.ml, w.acc, a.out_direct, a.len_bump);
}

template <int DK, int DV>
void launch_partial_nb(const Plan& pl, const PartialArgs& a, const WsView& w, hipStream_t s) {
  if (a.T > 1) {
    if (pl.blocks == 1)
      launch_partial<DK, DV, 1, true>(pl, a, w, s);
    else
      launch_partial<DK, DV, 2, true>(pl, a, w, s);
  } else {
    if (pl.blocks == 1)
      launch_partial<DK, DV, 1, false>(pl, a, w, s);
    else
      launch_partial<DK, DV, 2, false>(pl, a, w, s);
  }
}

// Query rows (h_q x T) as the plan's query-head count, or -1 if T is out of
// range or the product overflows.
int query_rows(int h_q, int T) {
  if (T < 1 || T > kMaxQueryRows) return -1;
  const int64_t r = (int64_t)h_q * T;
  return r > 2147483647 ? -1 : (int)r;
}

// Validation of everything but `out` in the documented order (NULL, shapes,
// alignment, scale, workspace), then the partial launch.  T query rows per
// head (T > 1: causal), planned as h_q*T query heads.
da_status partial_impl(const float* q, const float* K, const float* V, const float* k_new,
                       const float* v_new, const int32_t* len, float scale, int B, int h_q,
                       int h_kv, int n_max, int d_k, int d_v, int T, int chunk_rows,
                       void* workspace, size_t workspace_bytes, void* stream, const float* out,
                       bool need_out, Plan* out_plan, bool allow_direct = false) {
  if (!q || !K || !V || !len || (need_out && !out)) return DA_ERR_NULL;
  if ((k_new == nullptr) != (v_new == nullptr)) return DA_ERR_NULL;
  const int rows = query_rows(h_q, T);
  if (rows < 0 || h_q < 1) return DA_ERR_SHAPE;
  // Validated against the documented size (the plan for kMaxResident), run
  // with the device's own plan (never larger).
  Plan pl;
  da_status st = make_plan(B, rows, h_kv, n_max, d_k, d_v, chunk_rows, kMaxResident, &pl);
  if (st != DA_OK) return st;
  if (!aligned(q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(len, 4) ||
      !aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(out, 16))
    return DA_ERR_ALIGN;
  if (!std::isfinite(scale)) return DA_ERR_SCALE;
  if (!workspace || workspace_bytes < pl.bytes) return DA_ERR_WORKSPACE;
  if (!aligned(workspace, 16)) return DA_ERR_ALIGN;
  (void)make_plan(B, rows, h_kv, n_max, d_k, d_v, chunk_rows, device_resident(), &pl);
  if (out_plan) *out_plan = pl;

  const WsView w = view(pl, workspace);
  // K and V are written only when a fused append is asked for (k_new set).
  // Direct form: for a whole decode whose slabs are single chunks, or a
  // whole fused step in the two-wave direct form (the kernel then advances
  // len itself).
  float* direct = allow_direct && pl.single_chunk && (!k_new || direct_two_waves(pl, d_k, d_v))
                      ? const_cast<float*>(out)
                      : nullptr;
  int32_t* bump = direct && k_new ? const_cast<int32_t*>(len) : nullptr;
  const PartialArgs a{q, const_cast<float*>(K), const_cast<float*>(V), k_new, v_new, len,
                      scale * kLog2e, B, rows, h_kv, n_max, T, direct, bump};
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  if (d_k == 64 && d_v == 64) launch_partial_nb<64, 64>(pl, a, w, s);
  else if (d_k == 64 && d_v == 128) launch_partial_nb<64, 128>(pl, a, w, s);
  else if (d_k == 64 && d_v == 256) launch_partial_nb<64, 256>(pl, a, w, s);
  else if (d_k == 128 && d_v == 64) launch_partial_nb<128, 64>(pl, a, w, s);
  else if (d_k == 128 && d_v == 128) launch_partial_nb<128, 128>(pl, a, w, s);
  else if (d_k == 128 && d_v == 256) launch_partial_nb<128, 256>(pl, a, w, s);
  else if (d_k == 256 && d_v == 64) launch_partial_nb<256, 64>(pl, a, w, s);
  else if (d_k == 256 && d_v == 128) launch_partial_nb<256, 128>(pl, a, w, s);
  else launch_partial_nb<256, 256>(pl, a, w, s);
  return launch_status();
}

da_status merge_impl(float* out, int32_t* len_bump, int B, int h_q, int h_kv, int n_max,
                     int d_k, int d_v, int T, int chunk_rows, void* workspace,
                     size_t workspace_bytes, void* stream) {
  if (!out) return DA_ERR_NULL;
  const int rows = query_rows(h_q, T);
  if (rows < 0 || h_q < 1) return DA_ERR_SHAPE;
  Plan pl;
  da_status st = make_plan(B, rows, h_kv, n_max, d_k, d_v, chunk_rows, kMaxResident, &pl);
  if (st != DA_OK) return st;
  if (!aligned(out, 16) || !aligned(len_bump, 4)) return DA_ERR_ALIGN;
  if (!workspace || workspace_bytes < pl.bytes) return DA_ERR_WORKSPACE;
  if (!aligned(workspace, 16)) return DA_ERR_ALIGN;
  (void)make_plan(B, rows, h_kv, n_max, d_k, d_v, chunk_rows, device_resident(), &pl);

  const WsView w = view(pl, workspace);
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  const int heads_per_group = pl.blocks * kHeadsPerBlock;
  const dim3 grid((unsigned)pl.slabs * (unsigned)pl.merge_heads);
  if (d_v == 256)
    hipLaunchKernelGGL(decode_merge_kernel<256>, grid, dim3(kThreads), 0, s, out, w.ml, w.acc,
                       rows, h_kv, pl.head_groups, heads_per_group, pl.merge_heads, pl.J, w.cnt,
                       w.nvis, len_bump, n_max, T);
  else if (d_v == 64)
    hipLaunchKernelGGL(decode_merge_kernel<64>, grid, dim3(kThreads), 0, s, out, w.ml, w.acc,
                       rows, h_kv, pl.head_groups, heads_per_group, pl.merge_heads, pl.J, w.cnt,
                       w.nvis, len_bump, n_max, T);
  else
    hipLaunchKernelGGL(decode_merge_kernel<128>, grid, dim3(kThreads), 0, s, out, w.ml, w.acc,
                       rows, h_kv, pl.head_groups, heads_per_group, pl.merge_heads, pl.J, w.cnt,
                       w.nvis, len_bump, n_max, T);
  return launch_status();
}

// Zeroes n bytes (a multiple of 16) at p: the workspace counter reset, as a
// kernel rather than a memset so that it can be captured in a graph.
__global__ __launch_bounds__(kThreads) void clear_kernel(u4* __restrict__ p, size_t n16) {
  for (size_t e = (size_t)blockIdx.x * kThreads + threadIdx.x; e < n16;
       e += (size_t)gridDim.x * kThreads)
    p[e] = u4{0u, 0u, 0u, 0u};
}

da_status clear_words(void* p, size_t bytes, hipStream_t s) {
  const size_t n16 = bytes / 16;
  const unsigned grid = (unsigned)std::min<size_t>(1024, (n16 + kThreads - 1) / kThreads);
  (void)hipGetLastError();
  hipLaunchKernelGGL(clear_kernel, dim3(std::max(grid, 1u)), dim3(kThreads), 0, s,
                     static_cast<u4*>(p), n16);
  return launch_status();
}

}  // namespace

// ---------------------------------------------------------------------------
// Library-owned workspace for da_decode_attn_noalloc: a fixed array in device
// memory, one copy per GPU the library is loaded on, held until the process
// ends.  On the host, `scratch` names a host-side stand-in, never device
// memory: its device address is looked up per device (hipGetSymbolAddress)
// and only that address is passed to kernels.
// ---------------------------------------------------------------------------
static constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

static std::atomic<void*> g_scratch_ptr[kMaxDevices];

// Device address of this device's `scratch`, looked up on the first call on
// the device (with the device current) and kept; nullptr on a HIP error.
static void* scratch_address(int dev) {
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (p) return p;
  if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) {
    (void)hipGetLastError();
    return nullptr;
  }
  g_scratch_ptr[dev].store(p, std::memory_order_release);
  return p;
}

extern "C" {

const char* da_status_string(da_status status) {
  switch ((int)status) {
    case DA_OK: return "DA_OK";
    case DA_ERR_NULL: return "DA_ERR_NULL: a required pointer is NULL";
    case DA_ERR_SHAPE: return "DA_ERR_SHAPE: invalid sizes or chunk_rows";
    case DA_ERR_UNSUPPORTED: return "DA_ERR_UNSUPPORTED: head dimension not supported";
    case DA_ERR_ALIGN: return "DA_ERR_ALIGN: pointer not aligned";
    case DA_ERR_SCALE: return "DA_ERR_SCALE: scale is not finite";
    case DA_ERR_WORKSPACE: return "DA_ERR_WORKSPACE: workspace missing or too small";
    case DA_ERR_HIP: return "DA_ERR_HIP: HIP runtime error at launch";
    default: return "unknown da_status";
  }
}

size_t da_decode_workspace_bytes(int B, int h_q, int h_kv, int n_max, int d_k, int d_v) {
  return da_decode_workspace_bytes_ex(B, h_q, h_kv, n_max, d_k, d_v, 0);
}

size_t da_decode_workspace_counter_bytes(int B, int h_q, int h_kv, int n_max, int d_k,
                                         int d_v) {
  Plan pl;
  if (make_plan(B, h_q, h_kv, n_max, d_k, d_v, 0, kMaxResident, &pl) != DA_OK) return 0;
  return pl.counter_bytes;
}

da_status da_decode_workspace_reset(void* workspace, size_t workspace_bytes, int B, int h_q,
                                    int h_kv, int n_max, int d_k, int d_v, void* stream) {
  if (!workspace) return DA_ERR_NULL;
  Plan pl;
  const da_status st = make_plan(B, h_q, h_kv, n_max, d_k, d_v, 0, kMaxResident, &pl);
  if (st != DA_OK) return st;
  if (workspace_bytes < pl.counter_bytes) return DA_ERR_WORKSPACE;
  if (!aligned(workspace, 16)) return DA_ERR_ALIGN;
  return clear_words(workspace, pl.counter_bytes, static_cast<hipStream_t>(stream));
}

da_status da_decode_attn(const float* q, const float* K, const float* V, const int32_t* len,
                         float scale, float* out, int B, int h_q, int h_kv, int n_max,
                         int d_k, int d_v, void* workspace, size_t workspace_bytes,
                         void* stream) {
  return da_decode_multi_ex(q, K, V, len, scale, out, B, h_q, h_kv, n_max, d_k, d_v, 1, 0,
                            workspace, workspace_bytes, stream);
}

da_status da_decode_step(const float* q, float* K, float* V, const float* k_new,
                         const float* v_new, int32_t* len, float scale, float* out, int B,
                         int h_q, int h_kv, int n_max, int d_k, int d_v, void* workspace,
                         size_t workspace_bytes, void* stream) {
  return da_decode_multi_step(q, K, V, k_new, v_new, len, scale, out, B, h_q, h_kv, n_max,
                              d_k, d_v, 1, workspace, workspace_bytes, stream);
}

da_status da_decode_partial(const float* q, float* K, float* V, const float* k_new,
                            const float* v_new, const int32_t* len, float scale, int B,
                            int h_q, int h_kv, int n_max, int d_k, int d_v, void* workspace,
                            size_t workspace_bytes, void* stream) {
  return da_decode_partial_ex(q, K, V, k_new, v_new, len, scale, B, h_q, h_kv, n_max, d_k, d_v,
                              1, 0, workspace, workspace_bytes, stream);
}

da_status da_decode_merge(float* out, int32_t* len, int B, int h_q, int h_kv, int n_max,
                          int d_k, int d_v, void* workspace, size_t workspace_bytes,
                          void* stream) {
  return da_decode_merge_ex(out, len, B, h_q, h_kv, n_max, d_k, d_v, 1, 0, workspace,
                            workspace_bytes, stream);
}

da_status da_decode_multi(const float* q, const float* K, const float* V, const int32_t* len,
                          float scale, float* out, int B, int h_q, int h_kv, int n_max,
                          int d_k, int d_v, int T, void* workspace, size_t workspace_bytes,
                          void* stream) {
  return da_decode_multi_ex(q, K, V, len, scale, out, B, h_q, h_kv, n_max, d_k, d_v, T, 0,
                            workspace, workspace_bytes, stream);
}

da_status da_decode_multi_step(const float* q, float* K, float* V, const float* k_new,
                               const float* v_new, int32_t* len, float scale, float* out,
                               int B, int h_q, int h_kv, int n_max, int d_k, int d_v, int T,
                               void* workspace, size_t workspace_bytes, void* stream) {
  if (!k_new || !v_new) return DA_ERR_NULL;
  Plan pl;
  da_status st = partial_impl(q, K, V, k_new, v_new, len, scale, B, h_q, h_kv, n_max, d_k, d_v,
                              T, 0, workspace, workspace_bytes, stream, out, true, &pl, true);
  if (st != DA_OK) return st;
  if (direct_two_waves(pl, d_k, d_v)) return DA_OK;  // the direct form did the whole step
  return merge_impl(out, len, B, h_q, h_kv, n_max, d_k, d_v, T, pl.chunk_rows, workspace,
                    workspace_bytes, stream);
}

da_status da_kv_append_rows(float* K, float* V, const float* k_new, const float* v_new,
                            int32_t* len, int B, int h_kv, int n_max, int d_k, int d_v, int T,
                            void* stream) {
  if (!K || !V || !k_new || !v_new || !len) return DA_ERR_NULL;
  if (B < 1 || h_kv < 1 || n_max < 1 || d_k < 1 || d_v < 1 || T < 1 || T > kMaxQueryRows)
    return DA_ERR_SHAPE;
  if (d_k % 4 != 0 || d_v % 4 != 0) return DA_ERR_UNSUPPORTED;
  if ((int64_t)h_kv * T * (d_k / 4 + d_v / 4) > 2147483647) return DA_ERR_SHAPE;
  if (!aligned(K, 16) || !aligned(V, 16) || !aligned(k_new, 16) || !aligned(v_new, 16) ||
      !aligned(len, 4))
    return DA_ERR_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  hipLaunchKernelGGL(kv_append_kernel, dim3((unsigned)B), dim3(kThreads), 0, s, K, V, k_new,
                     v_new, len, h_kv, n_max, d_k, d_v, T);
  return launch_status();
}

da_status da_kv_append(float* K, float* V, const float* k_new, const float* v_new,
                       int32_t* len, int B, int h_kv, int n_max, int d_k, int d_v,
                       void* stream) {
  return da_kv_append_rows(K, V, k_new, v_new, len, B, h_kv, n_max, d_k, d_v, 1, stream);
}

// --- tuning and testing only: explicit segment size -------------------------

int da_decode_chunk_rows(int B, int h_q, int h_kv, int n_max, int d_k, int d_v) {
  Plan pl;
  if (make_plan(B, h_q, h_kv, n_max, d_k, d_v, 0, kMaxResident, &pl) != DA_OK) return 0;
  return pl.chunk_rows;
}

size_t da_decode_workspace_bytes_ex(int B, int h_q, int h_kv, int n_max, int d_k, int d_v,
                                    int chunk_rows) {
  Plan pl;
  if (make_plan(B, h_q, h_kv, n_max, d_k, d_v, chunk_rows, kMaxResident, &pl) != DA_OK)
    return 0;
  return pl.bytes;
}

da_status da_decode_multi_ex(const float* q, const float* K, const float* V,
                             const int32_t* len, float scale, float* out, int B, int h_q,
                             int h_kv, int n_max, int d_k, int d_v, int T, int chunk_rows,
                             void* workspace, size_t workspace_bytes, void* stream) {
  Plan pl;
  da_status st = partial_impl(q, K, V, nullptr, nullptr, len, scale, B, h_q, h_kv, n_max, d_k,
                              d_v, T, chunk_rows, workspace, workspace_bytes, stream, out, true,
                              &pl, true);
  if (st != DA_OK) return st;
  if (pl.single_chunk) return DA_OK;                  // the direct form wrote out
  return merge_impl(out, nullptr, B, h_q, h_kv, n_max, d_k, d_v, T, pl.chunk_rows, workspace,
                    workspace_bytes, stream);
}

da_status da_decode_partial_ex(const float* q, float* K, float* V, const float* k_new,
                               const float* v_new, const int32_t* len, float scale, int B,
                               int h_q, int h_kv, int n_max, int d_k, int d_v, int T,
                               int chunk_rows, void* workspace, size_t workspace_bytes,
                               void* stream) {
  return partial_impl(q, K, V, k_new, v_new, len, scale, B, h_q, h_kv, n_max, d_k, d_v, T,
                      chunk_rows, workspace, workspace_bytes, stream, nullptr, false, nullptr);
}

da_status da_decode_merge_ex(float* out, int32_t* len, int B, int h_q, int h_kv, int n_max,
                             int d_k, int d_v, int T, int chunk_rows, void* workspace,
                             size_t workspace_bytes, void* stream) {
  return merge_impl(out, len, B, h_q, h_kv, n_max, d_k, d_v, T, chunk_rows, workspace,
                    workspace_bytes, stream);
}

// --- no allocation: the library's own static workspace ----------------------

da_status da_decode_attn_noalloc(const float* q, const float* K, const float* V,
                                 const int32_t* len, float scale, float* out, int B, int h_q,
                                 int h_kv, int n_max, int d_k, int d_v, void* stream) {
  if (!q || !K || !V || !len || !out) return DA_ERR_NULL;
  Plan pl;
  da_status st = make_plan(B, h_q, h_kv, n_max, d_k, d_v, 0, kMaxResident, &pl);
  if (st != DA_OK) return st;
  if (pl.bytes > kScratchBytes) return DA_ERR_WORKSPACE;
  if (!aligned(q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(len, 4) ||
      !aligned(out, 16))
    return DA_ERR_ALIGN;
  if (!std::isfinite(scale)) return DA_ERR_SCALE;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return DA_ERR_HIP;
  }
  void* ws = scratch_address(dev);
  if (!ws) return DA_ERR_HIP;
  // The array keeps the last call's contents, possibly of other shapes: the
  // counter region of these shapes starts from zero.
  hipStream_t s = static_cast<hipStream_t>(stream);
  st = clear_words(ws, pl.counter_bytes, s);
  if (st != DA_OK) return st;
  return da_decode_multi_ex(q, K, V, len, scale, out, B, h_q, h_kv, n_max, d_k, d_v, 1, 0, ws,
                            kScratchBytes, stream);
}

}  // extern "C"
