// decode_attn.hip -- gfx950 kernels and C ABI for single-query decode
// attention over a KV cache (MHA/GQA/MQA) and the per-step KV append.
//
// Kernels
//   kv_append_kernel       eqs. (6)-(7): one bit-exact row copy per KV head,
//                          then len[b] += 1 (Proposition 2's (d_k+d_v)*4 B).
//   decode_partial_kernel  eqs. (1)-(3) over one split of one KV slab, for all
//                          query heads of its GQA group at once: the slab's
//                          rows are read from HBM once and feed every head of
//                          the group (the group caching of the GQA section).
//   decode_merge_kernel    combines split partials into the output row.
//
// Work decomposition of decode_partial_kernel
//   grid  (split p, KV head g x head group, batch b), 256 threads = 4 waves.
//   A workgroup owns rows [p*S, min((p+1)*S, n_b)) of slab (b, g); its waves
//   take 16-row tiles round-robin.  Each tile is two dense products on the
//   matrix cores (v_mfma_f32_16x16x4_f32, fp32 in and out):
//     scores  S[16 rows x 16 heads] = K_tile[16 x d_k] . Q^T[d_k x 16]
//     update  O^T[d_v x 16 heads]  += V_tile^T[d_v x 16] . P[16 x 16 heads]
//   with the online (running max / running sum) form of the softmax between
//   them, so the score vector never leaves registers.  Up to 16 query heads
//   ride in one product's columns; groups of 17..32 heads use two column
//   blocks over the same K/V registers, larger groups several head groups.
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
#include <cstdint>

#include "decode_attn.h"

typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int kWave = 64;
constexpr int kWaves = 4;
constexpr int kThreads = kWave * kWaves;
constexpr int kTileRows = 16;                        // rows per MFMA tile
constexpr int kHeadsPerBlock = 16;                   // heads per MFMA column block
constexpr int kSplitQuantum = kTileRows * kWaves;    // split sizes are multiples
constexpr int kMaxHeadBlocks = 2;                    // column blocks per workgroup
constexpr int kHeadsPerGroup = kHeadsPerBlock * kMaxHeadBlocks;
constexpr int kComputeUnits = 256;                   // MI355X
constexpr int kTargetWorkgroups = kComputeUnits * 8;
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

__device__ __forceinline__ int rows_used(int32_t len_b, int n_max) {
  return len_b < 0 ? 0 : (len_b > n_max ? n_max : len_b);
}

// ---------------------------------------------------------------------------
// KV append.  One workgroup per sequence; every thread reads len[b] before
// the barrier, thread 0 writes it after, so no thread can see the new value.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void kv_append_kernel(
    float* __restrict__ K, float* __restrict__ V,
    const float* __restrict__ k_new, const float* __restrict__ v_new,
    int32_t* __restrict__ len, int h_kv, int n_max, int d_k, int d_v) {
  const int b = blockIdx.x;
  const int32_t t = len[b];
  const bool room = t >= 0 && t < n_max;
  if (room) {
    const int ck = d_k / 4, cv = d_v / 4;            // 16-byte chunks per row
    const int per_head = ck + cv;
    const int total = h_kv * per_head;
    for (int c = threadIdx.x; c < total; c += blockDim.x) {
      const int g = c / per_head;
      const int w = c - g * per_head;
      const int64_t slab = (int64_t)b * h_kv + g;
      if (w < ck) {
        const u4* src = reinterpret_cast<const u4*>(k_new + slab * d_k) + w;
        u4* dst = reinterpret_cast<u4*>(K + (slab * n_max + t) * d_k) + w;
        *dst = *src;
      } else {
        const int wv = w - ck;
        const u4* src = reinterpret_cast<const u4*>(v_new + slab * d_v) + wv;
        u4* dst = reinterpret_cast<u4*>(V + (slab * n_max + t) * d_v) + wv;
        *dst = *src;
      }
    }
  }
  __syncthreads();
  if (room && threadIdx.x == 0) len[b] = t + 1;
}

// ---------------------------------------------------------------------------
// Split partials.
//   ws_ml  [B][h_q][P] float2 (running max in base-2 units, running sum)
//   ws_acc [B][h_q][P][DV]    unnormalised weighted sum of V rows
// ---------------------------------------------------------------------------
template <int DK, int DV, int NB>
struct Tile {
  f4 k[DK / 16];          // K rows: lane (i,k) holds row i, dims 16t+4k..+3
  f4 v[4][DV / 64];       // V rows: lane (i,k) holds row 4k+rho, dims 64c+4i..+3
};

template <int DK, int DV, int NB>
__device__ __forceinline__ void load_tile(Tile<DK, DV, NB>& T,
                                          const float* __restrict__ Ks,
                                          const float* __restrict__ Vs,
                                          int row0, int last_row, int i, int k) {
  const int rk = min(row0 + i, last_row);
#pragma unroll
  for (int t = 0; t < DK / 16; ++t)
    T.k[t] = load4(Ks + (int64_t)rk * DK + 16 * t + 4 * k);
#pragma unroll
  for (int rho = 0; rho < 4; ++rho) {
    const int rv = min(row0 + 4 * k + rho, last_row);
#pragma unroll
    for (int c = 0; c < DV / 64; ++c)
      T.v[rho][c] = load4(Vs + (int64_t)rv * DV + 64 * c + 4 * i);
  }
}

// One 16-row tile for NB column blocks of query heads: scores on the matrix
// cores, online softmax update, weighted-sum update on the matrix cores.
template <int DK, int DV, int NB>
__device__ __forceinline__ void process_tile(const Tile<DK, DV, NB>& T, int row0, int last_row,
                                             int k, int lane,
                                             const f4 (*__restrict__ sh_q)[DK / 16][kWave],
                                             float (&m_run)[NB], float (&l_run)[NB],
                                             f4 (&acc)[NB][DV / 64][4]) {
  // q is re-read from LDS for every tile rather than pinned in 32 VGPRs per
  // column block: the empty asm keeps the compiler from hoisting those reads
  // out of the tile loop, which would cost a second wave per SIMD.
  asm volatile("" ::: "memory");
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    f4 qb[DK / 16];
#pragma unroll
    for (int t = 0; t < DK / 16; ++t) qb[t] = sh_q[nb][t][lane];
    // Step I: s[row 4k+r][head i] for the tile's 16 rows (two independent
    // accumulation chains over the d_k/4 steps, added at the end).
    f4 s0 = f4{0.f, 0.f, 0.f, 0.f}, s1 = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < DK / 16; t += 2) {
      s0 = mfma_16x16x4(T.k[t].x, qb[t].x, s0);
      s1 = mfma_16x16x4(T.k[t + 1].x, qb[t + 1].x, s1);
      s0 = mfma_16x16x4(T.k[t].y, qb[t].y, s0);
      s1 = mfma_16x16x4(T.k[t + 1].y, qb[t + 1].y, s1);
      s0 = mfma_16x16x4(T.k[t].z, qb[t].z, s0);
      s1 = mfma_16x16x4(T.k[t + 1].z, qb[t + 1].z, s1);
      s0 = mfma_16x16x4(T.k[t].w, qb[t].w, s0);
      s1 = mfma_16x16x4(T.k[t + 1].w, qb[t + 1].w, s1);
    }
    f4 s = s0 + s1;
    // Rows past the split's end take no weight.
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (row0 + 4 * k + r > last_row) s[r] = -INFINITY;

    // Step II, online: running max over the 4 row groups of head i.
    float tmax = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    const float m_new = fmaxf(m_run[nb], tmax);
    const float alpha = fast_exp2(m_run[nb] - m_new);
    f4 pr;
    pr[0] = fast_exp2(s[0] - m_new);
    pr[1] = fast_exp2(s[1] - m_new);
    pr[2] = fast_exp2(s[2] - m_new);
    pr[3] = fast_exp2(s[3] - m_new);
    l_run[nb] = l_run[nb] * alpha + ((pr[0] + pr[1]) + (pr[2] + pr[3]));
    m_run[nb] = m_new;
#pragma unroll
    for (int c = 0; c < DV / 64; ++c)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[nb][c][e] *= alpha;

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

template <int DK, int DV, int NB>
__global__ __launch_bounds__(kThreads) void decode_partial_kernel(
    const float* __restrict__ q, const float* __restrict__ K,
    const float* __restrict__ V, const int32_t* __restrict__ len,
    float qscale, int h_q, int h_kv, int n_max, int split_rows, int P,
    int head_groups, float2* __restrict__ ws_ml, float* __restrict__ ws_acc) {
  const int p = blockIdx.x;
  const int g = blockIdx.y / head_groups;
  const int hgrp = blockIdx.y - g * head_groups;
  const int b = blockIdx.z;

  const int n_b = rows_used(len[b], n_max);
  const int row_begin = p * split_rows;
  if (row_begin >= n_b) return;                       // whole workgroup exits
  const int row_end = min(row_begin + split_rows, n_b);
  const int last_row = row_end - 1;

  const int G = h_q / h_kv;
  const int h_first = g * G + hgrp * (NB * kHeadsPerBlock);
  const int h_count = min(NB * kHeadsPerBlock, G - hgrp * (NB * kHeadsPerBlock));

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int i = lane & 15;
  const int k = lane >> 4;

  const int64_t slab = (int64_t)b * h_kv + g;
  const float* __restrict__ Ks = K + slab * n_max * DK;
  const float* __restrict__ Vs = V + slab * n_max * DV;

  // B operand of the score product, staged in LDS in register order: entry
  // [nb][t][lane (k, i)] = q of head nb*16+i at dims 16t+4k..+3, scaled into
  // base-2 units (zero for the padding heads of a partial column block).
  __shared__ f4 sh_q[NB][DK / 16][kWave];
  for (int e = threadIdx.x; e < NB * (DK / 16) * kWave; e += kThreads) {
    const int ln = e % kWave;
    const int t = (e / kWave) % (DK / 16);
    const int nb = e / (kWave * (DK / 16));
    const int hl = nb * kHeadsPerBlock + (ln & 15);
    f4 v = f4{0.f, 0.f, 0.f, 0.f};
    if (hl < h_count)
      v = load4(q + ((int64_t)b * h_q + h_first + hl) * DK + 16 * t + 4 * (ln >> 4)) * qscale;
    sh_q[nb][t][ln] = v;
  }
  __syncthreads();

  // Running state per column block; lane (k, i) belongs to head i.
  float m_run[NB], l_run[NB];
  f4 acc[NB][DV / 64][4];   // acc[nb][c][e][r] = O[dim 64c+16k+4r+e][head i]
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    m_run[nb] = -INFINITY;
    l_run[nb] = 0.f;
#pragma unroll
    for (int c = 0; c < DV / 64; ++c)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[nb][c][e] = f4{0.f, 0.f, 0.f, 0.f};
  }

  const int n_tiles = (row_end - row_begin + kTileRows - 1) / kTileRows;
  // Two register tiles in ping-pong: the next tile's loads are in flight
  // while the current one is on the matrix cores.
  Tile<DK, DV, NB> ta, tb;
  int tile = wave;
  if (tile < n_tiles) load_tile(ta, Ks, Vs, row_begin + tile * kTileRows, last_row, i, k);
  while (tile < n_tiles) {
    if (tile + kWaves < n_tiles)
      load_tile(tb, Ks, Vs, row_begin + (tile + kWaves) * kTileRows, last_row, i, k);
    process_tile<DK, DV, NB>(ta, row_begin + tile * kTileRows, last_row, k, lane, sh_q, m_run, l_run, acc);
    tile += kWaves;
    if (tile >= n_tiles) break;
    if (tile + kWaves < n_tiles)
      load_tile(ta, Ks, Vs, row_begin + (tile + kWaves) * kTileRows, last_row, i, k);
    process_tile<DK, DV, NB>(tb, row_begin + tile * kTileRows, last_row, k, lane, sh_q, m_run, l_run, acc);
    tile += kWaves;
  }

  // Row sums of head i are spread over the 4 row groups k.
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    l_run[nb] += __shfl_xor(l_run[nb], 16);
    l_run[nb] += __shfl_xor(l_run[nb], 32);
  }

  // Combine the 4 waves: waves 1..3 park their state in LDS in their own
  // register layout; wave 0 rescales and adds it lane by lane.
  __shared__ f4 sh_acc[kWaves - 1][NB][DV / 64][4][kWave];
  __shared__ float sh_m[kWaves - 1][NB][kWave];
  __shared__ float sh_l[kWaves - 1][NB][kWave];
  if (wave > 0) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      sh_m[wave - 1][nb][lane] = m_run[nb];
      sh_l[wave - 1][nb][lane] = l_run[nb];
#pragma unroll
      for (int c = 0; c < DV / 64; ++c)
#pragma unroll
        for (int e = 0; e < 4; ++e) sh_acc[wave - 1][nb][c][e][lane] = acc[nb][c][e];
    }
  }
  __syncthreads();
  if (wave != 0) return;

#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float M = m_run[nb];
#pragma unroll
    for (int w = 0; w < kWaves - 1; ++w) M = fmaxf(M, sh_m[w][nb][lane]);
    const float w0 = fast_exp2(m_run[nb] - M);
    float L = l_run[nb] * w0;
#pragma unroll
    for (int c = 0; c < DV / 64; ++c)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[nb][c][e] *= w0;
#pragma unroll
    for (int w = 0; w < kWaves - 1; ++w) {
      const float ww = fast_exp2(sh_m[w][nb][lane] - M);   // empty wave: exp2(-inf) = 0
      L += sh_l[w][nb][lane] * ww;
#pragma unroll
      for (int c = 0; c < DV / 64; ++c)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[nb][c][e] += sh_acc[w][nb][c][e][lane] * ww;
    }

    const int hl = nb * kHeadsPerBlock + i;
    if (hl < h_count) {
      const int64_t slot = ((int64_t)b * h_q + h_first + hl) * P + p;
      if (k == 0) ws_ml[slot] = make_float2(M, L);
      float* dst = ws_acc + slot * DV;
#pragma unroll
      for (int c = 0; c < DV / 64; ++c)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const f4 o = f4{acc[nb][c][0][r], acc[nb][c][1][r], acc[nb][c][2][r], acc[nb][c][3][r]};
          *reinterpret_cast<f4*>(dst + 64 * c + 16 * k + 4 * r) = o;
        }
    }
  }
}

// ---------------------------------------------------------------------------
// Merge: out[b,h,:] = sum_p 2^(m_p - M) acc_p / sum_p 2^(m_p - M) l_p.
// One workgroup per (b, h); thread = (16-byte column chunk, split subset).
// ---------------------------------------------------------------------------
template <int DV>
__global__ __launch_bounds__(kThreads) void decode_merge_kernel(
    const int32_t* __restrict__ len, float* __restrict__ out,
    const float2* __restrict__ ws_ml, const float* __restrict__ ws_acc,
    int h_q, int n_max, int split_rows, int P) {
  constexpr int kChunks = DV / 4;
  constexpr int kLanesP = kThreads / kChunks;       // splits visited in parallel
  const int bh = blockIdx.x;
  const int b = bh / h_q;
  const int n_b = rows_used(len[b], n_max);
  const int Pb = (n_b + split_rows - 1) / split_rows;
  const int ch = threadIdx.x % kChunks;
  const int ps = threadIdx.x / kChunks;
  float* orow = out + (int64_t)bh * DV;
  if (Pb == 0) {                                      // empty cache: zeros
    if (ps == 0) *reinterpret_cast<f4*>(orow + 4 * ch) = f4{0.f, 0.f, 0.f, 0.f};
    return;
  }
  const float2* ml = ws_ml + (int64_t)bh * P;
  const float* acc = ws_acc + (int64_t)bh * P * DV;

  __shared__ float sh_red[kThreads];
  float m = -INFINITY;
  for (int pp = threadIdx.x; pp < Pb; pp += kThreads) m = fmaxf(m, ml[pp].x);
  sh_red[threadIdx.x] = m;
  __syncthreads();
  for (int s = kThreads / 2; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) sh_red[threadIdx.x] = fmaxf(sh_red[threadIdx.x], sh_red[threadIdx.x + s]);
    __syncthreads();
  }
  const float M = sh_red[0];
  __syncthreads();

  f4 o = f4{0.f, 0.f, 0.f, 0.f};
  float L = 0.f;
  for (int pp = ps; pp < Pb; pp += kLanesP) {
    const float2 st = ml[pp];
    const float w = fast_exp2(st.x - M);
    L += st.y * w;
    o += load4(acc + (int64_t)pp * DV + 4 * ch) * w;
  }
  __shared__ f4 sh_o[kThreads];
  __shared__ float sh_l[kThreads];
  sh_o[threadIdx.x] = o;
  sh_l[threadIdx.x] = L;
  __syncthreads();
  if (ps == 0) {
    for (int j = 1; j < kLanesP; ++j) {
      o += sh_o[j * kChunks + ch];
      L += sh_l[j * kChunks + ch];
    }
    *reinterpret_cast<f4*>(orow + 4 * ch) = o / L;
  }
}

// ---------------------------------------------------------------------------
// Host side: validation, sizing, launches.
// ---------------------------------------------------------------------------
struct Plan {
  int split_rows;
  int P;             // splits per slab
  int head_groups;   // workgroups per KV head along the head axis
  int blocks;        // MFMA column blocks per workgroup (1 or 2)
  size_t ml_bytes;   // bytes of the (max, sum) section, padded to 256
  size_t bytes;      // total workspace bytes
};

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
bool dim_ok(int d) { return d == 64 || d == 128; }

int ceil_div(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

da_status check_shapes(int B, int h_q, int h_kv, int n_max, int d_k, int d_v) {
  if (B < 1 || h_q < 1 || h_kv < 1 || n_max < 1 || d_k < 1 || d_v < 1) return DA_ERR_SHAPE;
  if (h_q % h_kv != 0) return DA_ERR_SHAPE;
  if (B > 65535) return DA_ERR_SHAPE;
  const int G = h_q / h_kv;
  const int64_t groups = (int64_t)h_kv * ceil_div(G, kHeadsPerGroup);
  if (groups > 65535) return DA_ERR_SHAPE;
  if (!dim_ok(d_k) || !dim_ok(d_v)) return DA_ERR_UNSUPPORTED;
  return DA_OK;
}

int auto_split_rows(int B, int h_q, int h_kv, int n_max) {
  const int G = h_q / h_kv;
  const int64_t units = (int64_t)B * h_kv * ceil_div(G, kHeadsPerGroup);
  const int64_t rows = (units * n_max + kTargetWorkgroups - 1) / kTargetWorkgroups;
  int64_t s = ((rows + kSplitQuantum - 1) / kSplitQuantum) * kSplitQuantum;
  if (s < kSplitQuantum) s = kSplitQuantum;
  const int64_t cap = ((int64_t)n_max + kSplitQuantum - 1) / kSplitQuantum * kSplitQuantum;
  if (s > cap) s = cap;
  return (int)s;
}

da_status make_plan(int B, int h_q, int h_kv, int n_max, int d_k, int d_v, int split_rows,
                    Plan* plan) {
  da_status st = check_shapes(B, h_q, h_kv, n_max, d_k, d_v);
  if (st != DA_OK) return st;
  if (split_rows == 0) split_rows = auto_split_rows(B, h_q, h_kv, n_max);
  if (split_rows < kSplitQuantum || split_rows % kSplitQuantum != 0) return DA_ERR_SHAPE;
  const int G = h_q / h_kv;
  plan->split_rows = split_rows;
  plan->P = ceil_div(n_max, split_rows);
  plan->head_groups = ceil_div(G, kHeadsPerGroup);
  plan->blocks = G > kHeadsPerBlock ? 2 : 1;
  const size_t slots = (size_t)B * h_q * plan->P;
  plan->ml_bytes = (slots * sizeof(float2) + 255) / 256 * 256;
  plan->bytes = plan->ml_bytes + slots * (size_t)d_v * sizeof(float);
  return DA_OK;
}

da_status launch_status() {
  return hipGetLastError() == hipSuccess ? DA_OK : DA_ERR_HIP;
}

template <int DK, int DV, int NB>
void launch_partial(const Plan& pl, const float* q, const float* K, const float* V,
                    const int32_t* len, float qscale, int B, int h_q, int h_kv, int n_max,
                    float2* ml, float* acc, hipStream_t stream) {
  dim3 grid(pl.P, h_kv * pl.head_groups, B);
  hipLaunchKernelGGL((decode_partial_kernel<DK, DV, NB>), grid, dim3(kThreads), 0, stream,
                     q, K, V, len, qscale, h_q, h_kv, n_max, pl.split_rows, pl.P,
                     pl.head_groups, ml, acc);
}

template <int DK, int DV>
void launch_partial_nb(const Plan& pl, const float* q, const float* K, const float* V,
                       const int32_t* len, float qscale, int B, int h_q, int h_kv,
                       int n_max, float2* ml, float* acc, hipStream_t s) {
  if (pl.blocks == 1)
    launch_partial<DK, DV, 1>(pl, q, K, V, len, qscale, B, h_q, h_kv, n_max, ml, acc, s);
  else
    launch_partial<DK, DV, 2>(pl, q, K, V, len, qscale, B, h_q, h_kv, n_max, ml, acc, s);
}

da_status partial_impl(const float* q, const float* K, const float* V, const int32_t* len,
                       float scale, int B, int h_q, int h_kv, int n_max, int d_k, int d_v,
                       int split_rows, void* workspace, size_t workspace_bytes,
                       void* stream, Plan* out_plan) {
  if (!q || !K || !V || !len) return DA_ERR_NULL;
  Plan pl;
  da_status st = make_plan(B, h_q, h_kv, n_max, d_k, d_v, split_rows, &pl);
  if (st != DA_OK) return st;
  if (!aligned(q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(len, 4))
    return DA_ERR_ALIGN;
  if (!std::isfinite(scale)) return DA_ERR_SCALE;
  if (!workspace || workspace_bytes < pl.bytes) return DA_ERR_WORKSPACE;
  if (!aligned(workspace, 16)) return DA_ERR_ALIGN;
  if (out_plan) *out_plan = pl;

  float2* ml = static_cast<float2*>(workspace);
  float* acc = reinterpret_cast<float*>(static_cast<char*>(workspace) + pl.ml_bytes);
  const float qscale = scale * kLog2e;
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  if (d_k == 64 && d_v == 64) launch_partial_nb<64, 64>(pl, q, K, V, len, qscale, B, h_q, h_kv, n_max, ml, acc, s);
  else if (d_k == 64 && d_v == 128) launch_partial_nb<64, 128>(pl, q, K, V, len, qscale, B, h_q, h_kv, n_max, ml, acc, s);
  else if (d_k == 128 && d_v == 64) launch_partial_nb<128, 64>(pl, q, K, V, len, qscale, B, h_q, h_kv, n_max, ml, acc, s);
  else launch_partial_nb<128, 128>(pl, q, K, V, len, qscale, B, h_q, h_kv, n_max, ml, acc, s);
  return launch_status();
}

da_status merge_impl(const int32_t* len, float* out, int B, int h_q, int h_kv, int n_max,
                     int d_k, int d_v, int split_rows, const void* workspace,
                     size_t workspace_bytes, void* stream) {
  if (!len || !out) return DA_ERR_NULL;
  Plan pl;
  da_status st = make_plan(B, h_q, h_kv, n_max, d_k, d_v, split_rows, &pl);
  if (st != DA_OK) return st;
  if (!aligned(out, 16) || !aligned(len, 4)) return DA_ERR_ALIGN;
  if (!workspace || workspace_bytes < pl.bytes) return DA_ERR_WORKSPACE;
  if (!aligned(workspace, 16)) return DA_ERR_ALIGN;

  const float2* ml = static_cast<const float2*>(workspace);
  const float* acc =
      reinterpret_cast<const float*>(static_cast<const char*>(workspace) + pl.ml_bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  const dim3 grid((unsigned)B * (unsigned)h_q);
  if (d_v == 64)
    hipLaunchKernelGGL(decode_merge_kernel<64>, grid, dim3(kThreads), 0, s, len, out, ml, acc,
                       h_q, n_max, pl.split_rows, pl.P);
  else
    hipLaunchKernelGGL(decode_merge_kernel<128>, grid, dim3(kThreads), 0, s, len, out, ml,
                       acc, h_q, n_max, pl.split_rows, pl.P);
  return launch_status();
}

}  // namespace

extern "C" {

const char* da_status_string(int status) {
  switch (status) {
    case DA_OK: return "DA_OK";
    case DA_ERR_NULL: return "DA_ERR_NULL: a required pointer is NULL";
    case DA_ERR_SHAPE: return "DA_ERR_SHAPE: invalid sizes or split_rows";
    case DA_ERR_UNSUPPORTED: return "DA_ERR_UNSUPPORTED: head dimension not supported";
    case DA_ERR_ALIGN: return "DA_ERR_ALIGN: pointer not aligned";
    case DA_ERR_SCALE: return "DA_ERR_SCALE: scale is not finite";
    case DA_ERR_WORKSPACE: return "DA_ERR_WORKSPACE: workspace missing or too small";
    case DA_ERR_HIP: return "DA_ERR_HIP: HIP runtime error at launch";
    default: return "unknown da_status";
  }
}

int da_decode_split_rows(int B, int h_q, int h_kv, int n_max, int d_k, int d_v) {
  Plan pl;
  if (make_plan(B, h_q, h_kv, n_max, d_k, d_v, 0, &pl) != DA_OK) return 0;
  return pl.split_rows;
}

size_t da_decode_workspace_bytes(int B, int h_q, int h_kv, int n_max, int d_k, int d_v,
                                 int split_rows) {
  Plan pl;
  if (make_plan(B, h_q, h_kv, n_max, d_k, d_v, split_rows, &pl) != DA_OK) return 0;
  return pl.bytes;
}

da_status da_decode_partial(const float* q, const float* K, const float* V,
                            const int32_t* len, float scale, int B, int h_q, int h_kv,
                            int n_max, int d_k, int d_v, int split_rows, void* workspace,
                            size_t workspace_bytes, void* stream) {
  return partial_impl(q, K, V, len, scale, B, h_q, h_kv, n_max, d_k, d_v, split_rows,
                      workspace, workspace_bytes, stream, nullptr);
}

da_status da_decode_merge(const int32_t* len, float* out, int B, int h_q, int h_kv,
                          int n_max, int d_k, int d_v, int split_rows,
                          const void* workspace, size_t workspace_bytes, void* stream) {
  return merge_impl(len, out, B, h_q, h_kv, n_max, d_k, d_v, split_rows, workspace,
                    workspace_bytes, stream);
}

da_status da_decode_attn(const float* q, const float* K, const float* V, const int32_t* len,
                         float scale, float* out, int B, int h_q, int h_kv, int n_max,
                         int d_k, int d_v, int split_rows, void* workspace,
                         size_t workspace_bytes, void* stream) {
  if (!out) return DA_ERR_NULL;
  if (!aligned(out, 16)) {
    // Report the full validation order of the partial first (NULL before ALIGN).
    if (!q || !K || !V || !len) return DA_ERR_NULL;
    Plan pl;
    da_status st = make_plan(B, h_q, h_kv, n_max, d_k, d_v, split_rows, &pl);
    return st != DA_OK ? st : DA_ERR_ALIGN;
  }
  Plan pl;
  da_status st = partial_impl(q, K, V, len, scale, B, h_q, h_kv, n_max, d_k, d_v, split_rows,
                              workspace, workspace_bytes, stream, &pl);
  if (st != DA_OK) return st;
  return merge_impl(len, out, B, h_q, h_kv, n_max, d_k, d_v, pl.split_rows, workspace,
                    workspace_bytes, stream);
}

da_status da_kv_append(float* K, float* V, const float* k_new, const float* v_new,
                       int32_t* len, int B, int h_kv, int n_max, int d_k, int d_v,
                       void* stream) {
  if (!K || !V || !k_new || !v_new || !len) return DA_ERR_NULL;
  if (B < 1 || h_kv < 1 || n_max < 1 || d_k < 1 || d_v < 1 || B > 2147483647) return DA_ERR_SHAPE;
  if (d_k % 4 != 0 || d_v % 4 != 0) return DA_ERR_UNSUPPORTED;
  if ((int64_t)h_kv * (d_k / 4 + d_v / 4) > 2147483647) return DA_ERR_SHAPE;
  if (!aligned(K, 16) || !aligned(V, 16) || !aligned(k_new, 16) || !aligned(v_new, 16) ||
      !aligned(len, 4))
    return DA_ERR_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  hipLaunchKernelGGL(kv_append_kernel, dim3((unsigned)B), dim3(kThreads), 0, s, K, V, k_new,
                     v_new, len, h_kv, n_max, d_k, d_v);
  return launch_status();
}

}  // extern "C"
