// eb_backward.hip — backward of the pooled EmbeddingBag lookup with a fused
// row-wise optimizer update, for the AMD Instinct MI355X (gfx950).
//
// The paper's component benchmark profiles each submodule's forward and
// backward pass (Sec. III-A).  For sparse_arch (Sec. IV-A.2) the backward
// turns the gradient of the pooled output embeddings into a gradient for
// every table row that was read, and a sparse optimizer updates those rows.
// For row r of table t, with c_i = 1, w_i or 1/L (sum, weighted sum, mean):
//
//   G[d] = sum over positions i of table t with idx_i = r of
//          c_i * grad_out[b(i), Doff[t] + d]
//   SGD:               W[r] -= lr * G
//   row-wise Adagrad:  s[r] += mean_d G[d]^2;  W[r] -= lr * G / (sqrt(s[r]) + eps)
//
// Computed without atomics on data, and deterministically:
//   1. every position gets a 32-bit sort key (the table's key base + row) and
//      its bag id, and each table's first tile is found from the offsets;
//   2. (key, position) pairs are radix-sorted (rocPRIM): each row's
//      occurrences become one run, in position order, and each table's
//      positions stay inside that table's range of the sorted array;
//   3. each table's sorted range is cut into tiles of 64 or 128 positions; a
//      wavefront walks its tile's runs, pools each run's gradient rows with the
//      forward's 16-byte-slice gather and reduce-scatter (the gradient is an
//      fp32 "table" of B rows), and updates the run's table row; a run that
//      crosses a tile boundary leaves a partial sum in a per-tile slot;
//   4. a fix-up pass sums each crossing run's partials in a fixed order (set
//      by the run's length) and updates its row; each tile's info word (its
//      table, the key of its last run, whether that run goes on and whether
//      it started there) lets the pass find a run's tiles without the sorted
//      keys.
// Long runs (the hottest rows of a Zipf workload appear tens of thousands of
// times per batch) are thereby spread over as many wavefronts as they have
// tiles, and no wavefront waits for another.

#include <mutex>

#include <rocprim/device/device_radix_sort.hpp>
#include <rocprim/iterator/counting_iterator.hpp>

#include "eb_device.h"

// The static workspace of eb_backward_update_noalloc (see scratch_address).
constexpr size_t kScratchBytes = (size_t)EB_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace eb {
namespace {

// The (key, value) sort: onesweep passes of 9 bits with 1024-thread blocks of
// 8 items each.  rocPRIM's own choice for 32-bit pairs on this GPU takes 16
// items per thread, so a 1 M-pair sort runs as only 65 blocks per pass; with 8
// the backward step was 12% faster on 1 M lookups, 4% on 15 M and the same on
// 3 M (smaller blocks or fewer items were slower on the larger inputs).  Keys
// of up to 27 bits (tens of millions of rows) take three 9-bit passes instead
// of four 8-bit ones: 7-10% off the step there; 10-bit digits were slower.
using SortConfig = rocprim::radix_sort_config<
    rocprim::default_config, rocprim::default_config,
    rocprim::radix_sort_onesweep_config<rocprim::kernel_config<1024, 8>, rocprim::kernel_config<1024, 8>, 9,
                                        rocprim::block_radix_rank_algorithm::match>>;

constexpr uint32_t kNoKey = 0xFFFFFFFFu;  // larger than any key (keys fit below it)
constexpr uint8_t kTileContinues = 1;      // the tile's last run goes on into the next tile
constexpr uint8_t kTileOwnsRun = 2;        // ... and started in this tile: this tile finishes it
constexpr int kOptRowwiseAdagrad = 1;

struct BwdArgs {
  const TableMeta *meta;
  GatherCtx ctx;
  const void *indices;
  const void *offsets;
  const float *weights;
  const float *grad;      // grad_out [B, sum D]
  float *state;           // row-wise Adagrad state [sum R]
  uint32_t *keys;         // [N] sort keys by position
  int32_t *bag_of;        // [N] bag id by position
  const uint32_t *skeys;  // [N] sorted keys
  const uint32_t *spos;   // [N] in sorted order: positions, or bag ids when sorted_bags
  int32_t *tile_start;    // [T + 1] first tile of each table; [T] = number of tiles
  uint64_t *tile_info;    // [tiles] flags | table << 8 | key of the tile's last run << 32
  float *carry;           // [2 * tiles * max_dim]: slot 2w = head run partial, 2w+1 = tail run partial
  int64_t num_indices;
  int64_t grad_ld;        // sum D
  int32_t num_bags;
  int32_t batch;
  int32_t num_tables;
  int32_t idx64;
  int32_t coef;           // 0: c = 1, 1: c = w_i, 2: c = 1 / L
  int32_t sorted_bags;    // spos holds bag ids (no per-sample weights to look up)
  int32_t opt;
  float lr;
  float eps;
  int32_t tile_size;      // positions per tile (multiple of 64)
  int32_t max_dim;
  int32_t bags_per_wave;  // keys kernel: bags per wavefront
  int32_t groups_per_table;
  int32_t num_waves;
  int32_t xcd_remap;      // tiles kernel: XCD-contiguous workgroup order
};

__device__ __forceinline__ int64_t load_offset(const BwdArgs &a, int64_t g) {
  return a.idx64 ? static_cast<const int64_t *>(a.offsets)[g] : (int64_t) static_cast<const int32_t *>(a.offsets)[g];
}

__device__ __forceinline__ int64_t clamp_pos(int64_t p, int64_t lo, int64_t hi) {
  return p < lo ? lo : (p > hi ? hi : p);
}

// tiles of table t (its clamped position range cut into tile_size pieces)
__device__ __forceinline__ void table_range(const BwdArgs &a, int32_t t, int64_t &p0, int64_t &p1) {
  p0 = clamp_pos(load_offset(a, (int64_t)t * a.batch), 0, a.num_indices);
  p1 = clamp_pos(load_offset(a, (int64_t)(t + 1) * a.batch), p0, a.num_indices);
}

// Step 3a: first tile of every table, an exclusive scan of the tables' tile
// counts by one workgroup of NT threads (part: 2 * NT / 64 slots of LDS).
// Tile counts depend on the offsets alone, so the keys kernel's last
// workgroup runs this before its own positions.
template <int NT>
__device__ __forceinline__ void scan_tile_starts(const BwdArgs &a, int64_t *part) {
  constexpr int kWaves = NT / kWave;
  const int T = a.num_tables;
  const int tid = threadIdx.x;
  const int per = (T + NT - 1) / NT;
  const int t0 = tid * per < T ? tid * per : T;
  const int t1 = t0 + per < T ? t0 + per : T;
  int64_t sum = 0;
  for (int t = t0; t < t1; ++t) {
    int64_t p0, p1;
    table_range(a, t, p0, p1);
    sum += (p1 - p0 + a.tile_size - 1) / a.tile_size;
  }
  // exclusive scan of the per-thread sums: within each wavefront, then over
  // the wavefronts' totals
  const int lane = tid & (kWave - 1), wave = tid / kWave;
  int64_t incl = sum;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int64_t v = __shfl_up(incl, o);
    if (lane >= o) incl += v;
  }
  if (lane == kWave - 1) part[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    int64_t w = lane < kWaves ? part[lane] : 0;
#pragma unroll
    for (int o = 1; o < kWaves; o <<= 1) {
      const int64_t v = __shfl_up(w, o);
      if (lane >= o) w += v;
    }
    if (lane < kWaves) part[kWaves + lane] = w;  // inclusive totals of waves 0..lane
  }
  __syncthreads();
  int64_t run = incl - sum + (wave > 0 ? part[kWaves + wave - 1] : 0);
  if (tid == NT - 1) a.tile_start[T] = (int32_t)(run + sum);
  for (int t = t0; t < t1; ++t) {
    a.tile_start[t] = (int32_t)run;
    int64_t p0, p1;
    table_range(a, t, p0, p1);
    run += (p1 - p0 + a.tile_size - 1) / a.tile_size;
  }
}

// Keys and bag ids of positions [P0, P1) (bags g0 .. g0 + nb - 1, whose
// offsets lane j holds in my_off).  kKeyChunks chunks of 64 positions per
// round: every index load of a round is issued before its first key is
// stored, and none sits behind a branch (a position past P1 re-reads P1 - 1),
// so a round costs one memory round trip.  Returns whether this lane saw an
// index outside the table.
template <typename IT>
__device__ __forceinline__ bool key_positions(const BwdArgs &a, const TableMeta &m, int64_t P0, int64_t P1,
                                              int64_t my_off, int nb, int32_t g0) {
  constexpr int kKeyChunks = 4;
  const int lane = threadIdx.x & (kWave - 1);
  const IT *idx = static_cast<const IT *>(a.indices);
  bool oob = false;
  for (int64_t c = P0; c < P1; c += kKeyChunks * kWave) {
    int64_t r[kKeyChunks];
#pragma unroll
    for (int u = 0; u < kKeyChunks; ++u) {
      const int64_t p = c + u * kWave + lane;
      r[u] = (int64_t)__builtin_nontemporal_load(idx + (p < P1 ? p : P1 - 1));
    }
#pragma unroll
    for (int u = 0; u < kKeyChunks; ++u) {
      const int64_t p = c + u * kWave + lane;
      if (p < P1) {
        int j = 0;
        for (int jj = 1; jj < nb; ++jj)
          if (readlane64(my_off, jj) <= p) j = jj;
        const bool ok = r[u] >= 0 && r[u] < m.num_rows;
        oob |= !ok;
        a.keys[p] = m.key_base + (ok ? (uint32_t)r[u] : (uint32_t)m.num_rows);
        a.bag_of[p] = g0 + j;
      }
    }
  }
  return oob;
}

// Step 1: sort key and bag id of every position.  A wavefront takes a run of
// consecutive bags of one table and walks their positions 64 at a time (the
// same work map as the forward).  An index outside its table gets the table's
// sentinel key (one past its last row), which sorts after the table's rows
// and is skipped later.
__global__ __launch_bounds__(kBlock) void eb_bwd_keys_kernel(BwdArgs a) {
  if (blockIdx.x == gridDim.x - 1) {
    // every thread of the workgroup, before any wavefront can leave
    __shared__ int64_t part[2 * kWavesPerBlock];
    scan_tile_starts<kBlock>(a, part);
  }
  const int32_t wid = (int32_t)blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  if (wid >= a.num_waves) return;
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t t = wid / a.groups_per_table;
  const int32_t b0 = (wid - t * a.groups_per_table) * a.bags_per_wave;
  const int nb = (a.batch - b0) < a.bags_per_wave ? (a.batch - b0) : a.bags_per_wave;
  const int32_t g0 = t * a.batch + b0;
  const TableMeta m = a.meta[t];
  const int64_t N = a.num_indices;

  int64_t raw = 0;
  if (lane <= nb) raw = load_offset(a, g0 + lane);
  // report a broken partition (checked mode); positions are clamped into [0, N)
  const int64_t nxt = __shfl_down(raw, 1);
  bool bad = lane < nb && (raw < 0 || nxt < raw || nxt > N);
  bad |= lane == 0 && g0 == 0 && raw != 0;
  bad |= lane == nb && g0 + nb == a.num_bags && raw != N;
  if (__ballot(bad)) {
    if (lane == 0) atomicOr(a.ctx.err, kErrOffsets);
  }
  const int64_t my_off = clamp_pos(raw, 0, N);
  const int64_t P0 = readlane64(my_off, 0);
  const int64_t P1 = readlane64(my_off, nb);
  const bool oob = a.idx64 ? key_positions<int64_t>(a, m, P0, P1, my_off, nb, g0)
                           : key_positions<int32_t>(a, m, P0, P1, my_off, nb, g0);
  if (__ballot(oob)) {
    if (lane == 0) atomicOr(a.ctx.err, kErrIndex);
  }
}

// table owning tile w: the last table whose first tile is <= w (empty tables
// own no tile and are skipped)
__device__ __forceinline__ int32_t table_of_tile(const BwdArgs &a, int32_t w) {
  int32_t lo = 0, hi = a.num_tables - 1;
  while (lo < hi) {
    const int32_t mid = (lo + hi + 1) / 2;
    if (a.tile_start[mid] <= w) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// Sum of x over the 64 lanes (fixed butterfly order).
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) x += __shfl_xor(x, o);
  return x;
}

// Table rows, the optimizer state and the carry slots are plain device
// memory, addressed in the global address space so that their accesses compile
// to global instructions.  A flat access also counts as an LDS access: the wait
// before the next cross-lane shuffle would wait for it too, and a row read
// ahead of a gradient gather would no longer overlap the gather.
typedef EB_GLOBAL unsigned char growb;
typedef EB_GLOBAL float gf32;
typedef EB_GLOBAL _Float16 gf16;
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ growb *row_bytes(const TableMeta &m, int64_t row) {
  return (growb *)m.data + (uint64_t)row * m.row_stride;
}

__device__ __forceinline__ gf32 *state_of(const BwdArgs &a, const TableMeta &m, int64_t row) {
  return (gf32 *)a.state + m.state_base + row;
}

// K = 1, 2 or 4 consecutive values of a row of type TDT from column col (a
// multiple of K, so the access is aligned to its size), in one access.
template <int TDT, int K>
__device__ __forceinline__ void load_vals(growb *base, int col, float (&w)[K]) {
  static_assert(K == 1 || K == 2 || K == 4, "one access holds 1, 2 or 4 values");
  if constexpr (TDT == kF32) {
    gf32 *p = (gf32 *)base + col;
    if constexpr (K == 4) {
      const f32x4 v = *(EB_GLOBAL f32x4 *)p;
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = v[i];
    } else if constexpr (K == 2) {
      const f32x2 v = *(EB_GLOBAL f32x2 *)p;
      w[0] = v[0];
      w[1] = v[1];
    } else {
      w[0] = *p;
    }
  } else {
    gf16 *p = (gf16 *)base + col;
    if constexpr (K == 4) {
      const f16x4 v = *(EB_GLOBAL f16x4 *)p;
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = (float)v[i];
    } else if constexpr (K == 2) {
      const f16x2 v = *(EB_GLOBAL f16x2 *)p;
      w[0] = (float)v[0];
      w[1] = (float)v[1];
    } else {
      w[0] = (float)*p;
    }
  }
}

// The store matching load_vals (fp16 rows round to nearest).
template <int TDT, int K>
__device__ __forceinline__ void store_vals(growb *base, int col, const float (&w)[K]) {
  static_assert(K == 1 || K == 2 || K == 4, "one access holds 1, 2 or 4 values");
  if constexpr (TDT == kF32) {
    gf32 *p = (gf32 *)base + col;
    if constexpr (K == 4) *(EB_GLOBAL f32x4 *)p = f32x4{w[0], w[1], w[2], w[3]};
    else if constexpr (K == 2) *(EB_GLOBAL f32x2 *)p = f32x2{w[0], w[1]};
    else *p = w[0];
  } else {
    gf16 *p = (gf16 *)base + col;
    if constexpr (K == 4) {
      *(EB_GLOBAL f16x4 *)p = f16x4{(_Float16)w[0], (_Float16)w[1], (_Float16)w[2], (_Float16)w[3]};
    } else if constexpr (K == 2) {
      *(EB_GLOBAL f16x2 *)p = f16x2{(_Float16)w[0], (_Float16)w[1]};
    } else {
      *p = (_Float16)w[0];
    }
  }
}

// The values a row update reads, loaded ahead of the gather that produces
// the row's gradient: the lane's K table values and the Adagrad state.
template <int TDT, int K>
struct RowPrefetch {
  float w[K];
  float s;
};

template <int TDT, int K>
__device__ __forceinline__ RowPrefetch<TDT, K> prefetch_row(const TableMeta &m, const BwdArgs &a, int64_t row, bool own,
                                                           int col) {
  RowPrefetch<TDT, K> p;
  p.s = a.opt == kOptRowwiseAdagrad ? *state_of(a, m, row) : 0.0f;
#pragma unroll
  for (int i = 0; i < K; ++i) p.w[i] = 0.0f;
  if (own) load_vals<TDT, K>(row_bytes(m, row), col, p.w);
  return p;
}

// Optimizer step on row `row` of table m.  Lane holds K gradient values for
// columns [col, col + K) when `own`; the columns of all owning lanes cover
// the row exactly once.  `p` holds the row's values read beforehand.
template <int TDT, int K>
__device__ __forceinline__ void apply_update(const TableMeta &m, const BwdArgs &a, int64_t row, const float (&g)[K],
                                             bool own, int col, const RowPrefetch<TDT, K> &p) {
  float scale = a.lr;
  if (a.opt == kOptRowwiseAdagrad) {
    float sq = 0.0f;
    if (own) {
#pragma unroll
      for (int i = 0; i < K; ++i) sq = fmaf(g[i], g[i], sq);
    }
    sq = wave_sum(sq);
    const float s_new = p.s + sq / (float)m.dim;
    scale = a.lr / (sqrtf(s_new) + a.eps);
    if ((threadIdx.x & (kWave - 1)) == 0) *state_of(a, m, row) = s_new;
  }
  if (own) {
    float nw[K];
#pragma unroll
    for (int i = 0; i < K; ++i) nw[i] = fmaf(-scale, g[i], p.w[i]);
    store_vals<TDT, K>(row_bytes(m, row), col, nw);
  }
}

// Complete runs inside one chunk, several at once: the runs that start at
// heads h_0 < ... < h_nruns of the chunk (run k is [h_k, h_k+1)) go to lane
// groups of LPRS lanes, one run per group, G = 64 / LPRS runs per round.  A
// group walks its run's entries in order (P 16-byte loads per lane per
// gradient row), then applies the optimizer step to the run's row itself:
// no cross-group reduction, and one memory round trip per round of G runs.
// A gradient row of 16 or more 16-byte slices is held by half as many lanes,
// two slices each: twice the runs per round, for the same registers that the
// widest row already takes.
template <int TDT, int LPR_NAT>
__device__ __forceinline__ void short_runs(const BwdArgs &a, const TableMeta &m, const TableMeta &gm, const Chunk &ch,
                                           uint32_t key, uint64_t hs, int nruns, int *starts) {
  constexpr int LPRS = LPR_NAT >= 16 ? LPR_NAT / 2 : LPR_NAT;
  constexpr int P = LPR_NAT / LPRS;
  constexpr int G = kWave / LPRS;
  constexpr int US = P >= 2 ? 2 : 4;
  constexpr int NV = 4 * P;
  const int lane = threadIdx.x & (kWave - 1);
  const int grp = lane / LPRS, sub = lane % LPRS;
  const uint32_t kmin = m.key_base, sentinel = m.key_base + (uint32_t)m.num_rows;
  // position of the head of each rank (rank = heads below it)
  if ((hs >> lane) & 1ull) starts[__builtin_popcountll(hs & ((1ull << lane) - 1ull))] = lane;
  __builtin_amdgcn_wave_barrier();
  const int colb0 = sub * 16 * P;
  for (int r0 = 0; r0 < nruns; r0 += G) {
    const int k = r0 + grp;
    const bool active = k < nruns;
    const int st = active ? starts[k] : 0;
    const int len = active ? starts[k + 1] - st : 0;
    const uint32_t rkey = (uint32_t)__shfl((int)key, st & (kWave - 1));
    const bool valid = active && rkey >= kmin && rkey < sentinel;
    const int64_t row = valid ? (int64_t)(rkey - kmin) : 0;
    int maxlen = len;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) maxlen = max(maxlen, __shfl_xor(maxlen, o));
    // the row's values and state, read before the gradient gather
    float wv[NV];
    float s_old = 0.0f;
#pragma unroll
    for (int i = 0; i < NV; ++i) wv[i] = 0.0f;
    const int col0 = colb0 / 4;
    if (valid) {
      if (a.opt == kOptRowwiseAdagrad) s_old = *state_of(a, m, row);
      growb *base = row_bytes(m, row);
#pragma unroll
      for (int pp = 0; pp < P; ++pp) {
        // dim is a multiple of 4: four columns are all in the row or all past it
        if (col0 + 4 * pp < m.dim) {
          float t4[4];
          load_vals<TDT, 4>(base, col0 + 4 * pp, t4);
#pragma unroll
          for (int i = 0; i < 4; ++i) wv[4 * pp + i] = t4[i];
        }
      }
    }
    float acc[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) acc[i] = 0.0f;
    for (int u = 0; u < maxlen; u += US) {
      u32x4 v[US][P];
      float c[US];
#pragma unroll
      for (int q = 0; q < US; ++q) {
        const int e = st + u + q;
        const uint32_t b = (uint32_t)__shfl((int)ch.row, e & (kWave - 1));
        c[q] = __shfl(ch.w, e & (kWave - 1));
        const bool ok = valid && (u + q < len) && b != kBadRow;
        gbyte *pr = ok ? (gbyte *)gm.data + (uint64_t)b * gm.row_stride : (gbyte *)a.ctx.zero;
#pragma unroll
        for (int pp = 0; pp < P; ++pp) {
          const int cb = colb0 + 16 * pp;
          v[q][pp] = load_slice<kF32>((cb < gm.code_bytes ? pr : (gbyte *)a.ctx.zero) + cb);
        }
      }
#pragma unroll
      for (int q = 0; q < US; ++q) {
#pragma unroll
        for (int pp = 0; pp < P; ++pp) {
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[4 * pp + i] = fmaf(c[q], __uint_as_float(v[q][pp][i]), acc[4 * pp + i]);
        }
      }
    }
    float scale = a.lr;
    if (a.opt == kOptRowwiseAdagrad) {
      float sq = 0.0f;
#pragma unroll
      for (int i = 0; i < NV; ++i) sq = fmaf(acc[i], acc[i], sq);  // zero past the row's end
#pragma unroll
      for (int o = 1; o < LPRS; o <<= 1) sq += __shfl_xor(sq, o);
      const float s_new = s_old + sq / (float)m.dim;
      scale = a.lr / (sqrtf(s_new) + a.eps);
      if (valid && sub == 0) *state_of(a, m, row) = s_new;
    }
    if (valid) {
      growb *base = row_bytes(m, row);
#pragma unroll
      for (int pp = 0; pp < P; ++pp) {
        if (col0 + 4 * pp < m.dim) {
          float t4[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) t4[i] = fmaf(-scale, acc[4 * pp + i], wv[4 * pp + i]);
          store_vals<TDT, 4>(base, col0 + 4 * pp, t4);
        }
      }
    }
  }
  __builtin_amdgcn_wave_barrier();
}

// Step 3b: pool the runs of one tile and update their rows (or leave
// partials).  LPR lanes hold one fp32 gradient row of 4*dim bytes.
template <int TDT, int LPR>
__device__ __forceinline__ void tile_body(const BwdArgs &a, const TableMeta &m, int32_t t, int32_t w, int32_t k,
                                          int *starts) {
  using R = Reduce<kF32, LPR>;
  constexpr int KEEP = R::KEEP;
  const int lane = threadIdx.x & (kWave - 1);
  int64_t p0, p1;
  table_range(a, t, p0, p1);
  const int64_t s = p0 + (int64_t)k * a.tile_size;
  const int64_t e = s + a.tile_size < p1 ? s + a.tile_size : p1;
  if (s >= e) return;
  const uint32_t before = s > p0 ? a.skeys[s - 1] : kNoKey;
  const uint32_t after = e < p1 ? a.skeys[e] : kNoKey;
  const uint32_t key_last = a.skeys[e - 1];
  const uint32_t kmin = m.key_base, sentinel = m.key_base + (uint32_t)m.num_rows;
  if (lane == 0) {
    const bool cont = after != kNoKey && after == key_last;
    const bool owns = cont && key_last != before && key_last < sentinel && key_last >= kmin;
    a.tile_info[w] = (uint64_t)((cont ? kTileContinues : 0) | (owns ? kTileOwnsRun : 0)) | ((uint64_t)t << 8) |
                     ((uint64_t)key_last << 32);
  }

  // the gradient rows of this table as an fp32 table of B rows
  TableMeta gm = m;
  gm.data = reinterpret_cast<const unsigned char *>(a.grad + m.out_col);
  gm.row_stride = (uint32_t)(a.grad_ld * 4);
  gm.num_rows = a.batch;
  gm.code_bytes = 4 * m.dim;
  const int colb = (lane % LPR) * 16;
  const bool colok = colb < gm.code_bytes;
  const int col = colb / 4 + R::first_value(lane);
  const bool own = R::stores(lane) && colok;

  float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  bool first_run = true;
  // Values of the row the current run will update, read when the run starts
  // (a run that crossed into this tile, or goes on past it, updates nothing
  // here); no other wavefront writes that row during this launch.
  RowPrefetch<TDT, KEEP> pre;
  auto start_run = [&](uint32_t rkey) {
    const bool valid = rkey >= kmin && rkey < sentinel;
    if (valid && !(first_run && rkey == before) && rkey != after)
      pre = prefetch_row<TDT, KEEP>(m, a, (int64_t)(rkey - kmin), own, col);
  };
  // Finish the run with key rkey whose terms are all in acc: update its row,
  // or leave a partial when it crosses a tile boundary.
  auto finish = [&](uint32_t rkey, bool reaches_end) {
    const bool valid = rkey >= kmin && rkey < sentinel;
    const bool started_before = first_run && rkey == before;
    const bool continues_after = reaches_end && rkey == after;
    if (valid) {
      R::run(acc);
      float gk[KEEP];
#pragma unroll
      for (int i = 0; i < KEEP; ++i) gk[i] = acc[i];
      if (!started_before && !continues_after) {
        apply_update<TDT, KEEP>(m, a, (int64_t)(rkey - kmin), gk, own, col, pre);
      } else if (own) {
        gf32 *slot = (gf32 *)a.carry + ((int64_t)2 * w + (started_before ? 0 : 1)) * a.max_dim;
        store_vals<kF32, KEEP>((growb *)slot, col, gk);
      }
    }
    first_run = false;
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = 0.0f;
  };
  bool pending = false;  // acc holds a run that reached the end of the previous chunk
  uint32_t pending_key = kNoKey;
  uint32_t prev_last = before;
  for (int64_t c = s; c < e; c += kWave) {
    const int n = (int)((e - c) < kWave ? (e - c) : kWave);
    const bool last_chunk = c + kWave >= e;
    uint32_t key = kNoKey;
    Chunk ch;
    ch.row = kBadRow;
    ch.w = 0.0f;
    ch.n = n;
    if (lane < n) {
      key = a.skeys[c + lane];
      // unweighted pooling sorts bag ids with the keys; weighted pooling sorts
      // positions (the weight is per position) and looks the bag up
      const uint32_t sv = a.spos[c + lane];
      const uint32_t pos = sv;
      const int32_t g = a.sorted_bags ? (int32_t)sv : a.bag_of[pos];
      const int64_t b = (int64_t)g - (int64_t)t * a.batch;
      if (key >= kmin && key < sentinel && b >= 0 && b < a.batch) {
        ch.row = (uint32_t)b;
        if (a.coef == 1) {
          ch.w = a.weights[pos];
        } else if (a.coef == 2) {
          const int64_t L = load_offset(a, g + 1) - load_offset(a, g);
          ch.w = L > 0 ? 1.0f / (float)L : 0.0f;
        } else {
          ch.w = 1.0f;
        }
      }
    }
    const uint32_t up = (uint32_t)__shfl_up((int)key, 1);
    const uint32_t prev = lane == 0 ? prev_last : up;
    const uint64_t heads = __ballot(lane < n && key != prev);
    // a run that ended exactly at the previous chunk's end
    if (pending && (heads & 1ull)) {
      finish(pending_key, false);
      pending = false;
    }
    int a0 = 0;
    if (!(heads & 1ull)) {
      // the chunk opens inside a run: the pending one, or the tile's first
      // run when it started in the previous tile
      const int z = heads ? (int)__builtin_ctzll(heads) : n;
      const uint32_t rkey = __builtin_amdgcn_readlane(key, 0);
      if (!pending) start_run(rkey);
      if (a.coef == 0) gather_range<kF32, LPR, false>(gm, a.ctx, ch, 0, z, acc, colb, colok);
      else gather_range<kF32, LPR, true>(gm, a.ctx, ch, 0, z, acc, colb, colok);
      if (z < n || last_chunk) {
        finish(rkey, z == n);
        pending = false;
      } else {
        pending = true;
        pending_key = rkey;
      }
      a0 = z;
    }
    if (a0 < n) {
      // runs starting at heads: all but the last are complete inside this
      // chunk and are updated here, several at once
      const uint64_t hs = heads;
      const int nheads = __builtin_popcountll(hs);
      if (nheads > 1) {
        short_runs<TDT, LPR>(a, m, gm, ch, key, hs, nheads - 1, starts);
        first_run = false;
      }
      const int hl = 63 - __builtin_clzll(hs);
      const uint32_t rkey = __builtin_amdgcn_readlane(key, hl);
      start_run(rkey);
      if (a.coef == 0) gather_range<kF32, LPR, false>(gm, a.ctx, ch, hl, n - hl, acc, colb, colok);
      else gather_range<kF32, LPR, true>(gm, a.ctx, ch, hl, n - hl, acc, colb, colok);
      if (last_chunk) {
        finish(rkey, true);
        pending = false;
      } else {
        pending = true;
        pending_key = rkey;
      }
    }
    prev_last = __builtin_amdgcn_readlane(key, n - 1);
  }
}

#define EB_BWD_LPR(LOG2)                                                        \
  case LOG2:                                                                    \
    tile_body<TDT, (1 << (LOG2))>(a, m, t, w, w - a.tile_start[t], starts);     \
    break;

// Wavefronts per tiles-kernel workgroup.  A tile's time varies several-fold
// with its runs (a chunk of single-occurrence rows takes many rounds, a piece
// of a hot row's run one gather); one-wavefront workgroups let a finished
// wavefront's slot take the next tile at once, where a four-wavefront
// workgroup waits for a free slot on every SIMD (measured 3-5% faster).
constexpr int kTileWaves = 1;

// Tiles are numbered table by table; with XCD-contiguous workgroup order each
// XCD walks one eighth of the tables, so its L2 keeps those tables' gradient
// rows (B x D fp32 per table, re-read by every run of the table) instead of
// all eight XCDs pulling the same table's gradient through the fabric.
template <int TDT, int LOG2>
__global__ __launch_bounds__(kWave * kTileWaves) void eb_bwd_tiles_kernel(BwdArgs a) {
  const uint32_t blk = a.xcd_remap ? xcd_contiguous(blockIdx.x, gridDim.x) : blockIdx.x;
  const int32_t w = (int32_t)blk * kTileWaves + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  if (w >= a.tile_start[a.num_tables]) return;
  const int32_t t = table_of_tile(a, w);
  const TableMeta m = a.meta[t];
  if (m.kind / 8 != TDT) return;
  __shared__ int run_starts[kTileWaves][kWave + 1];
  int *starts = run_starts[threadIdx.x / kWave];
  if constexpr (LOG2 >= 0) {
    tile_body<TDT, (1 << LOG2)>(a, m, t, w, w - a.tile_start[t], starts);
  } else {
    switch (log2_lanes_per_row(4 * m.dim)) {
      EB_BWD_LPR(0) EB_BWD_LPR(1) EB_BWD_LPR(2) EB_BWD_LPR(3) EB_BWD_LPR(4) EB_BWD_LPR(5) EB_BWD_LPR(6)
      default:
        break;
    }
  }
}

#undef EB_BWD_LPR

// Step 4: a run that starts in tile w and goes on past it: sum its partial
// from tile w and the head partials of the tiles it covers, in tile order,
// then update its row.  The run's last tile is found 64 tiles at a time (one
// per lane); the partials are summed with eight loads in flight.  Lane l
// handles columns [4l, 4l + 4).
template <int TDT>
__global__ __launch_bounds__(kBlock) void eb_bwd_fixup_kernel(BwdArgs a) {
  const int32_t w = (int32_t)blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int32_t total = a.tile_start[a.num_tables];
  if (w >= total) return;
  // every tile below `total` holds at least one position, so its info word
  // was written by this step's tiles kernel
  const uint64_t info = a.tile_info[w];
  if (!(info & kTileOwnsRun)) return;
  const int32_t t = (int32_t)((info >> 8) & 0xFFFFFFu);
  const uint32_t key = (uint32_t)(info >> 32);
  const TableMeta m = a.meta[t];
  if (m.kind / 8 != TDT) return;
  const int lane = threadIdx.x & (kWave - 1);
  // Row columns are held 4 per lane by L lanes (L = the next power of two
  // >= dim/4); the wavefront's G = 64/L lane groups add the partials of
  // tiles w+1+gi, w+1+gi+G, ... (group gi), and group 0 then adds the
  // groups' sums in group order.  The order of the sum is fixed by the run's
  // length alone, so results are reproducible.
  int L = 1;
  while (L < kWave && 4 * L < m.dim) L <<= 1;
  const int G = kWave / L;
  const int gi = lane / L;
  const int col = 4 * (lane % L);
  const bool cols = col < m.dim;
  const bool own = cols && gi == 0;
  constexpr int kBatch = 8;
  auto head = [&](int32_t tile) {  // partial of the run that enters `tile`
    return *(EB_GLOBAL const f32x4 *)((gf32 *)a.carry + ((int64_t)2 * tile) * a.max_dim + col);
  };
  // Issued before the run's end is known: the row and its state, this
  // tile's partial and that of tile w + 1, which is always in the run.
  const RowPrefetch<TDT, 4> pre = prefetch_row<TDT, 4>(m, a, (int64_t)(key - m.key_base), own, col);
  f32x4 tail = {0.0f, 0.0f, 0.0f, 0.0f}, next = {0.0f, 0.0f, 0.0f, 0.0f};
  if (own) {
    tail = *(EB_GLOBAL const f32x4 *)((gf32 *)a.carry + ((int64_t)2 * w + 1) * a.max_dim + col);
    next = head(w + 1);
  }
  // The run's last tile kend: every tile of the run but its last goes on
  // with the same key, and no tile after it does (the keys are sorted, and a
  // table's last tile never goes on), so it is the first tile after w that
  // fails the test.  Most runs end within the next 64 tiles (one load per
  // lane); longer ones are searched coarse to fine: tiles 64 apart, then the
  // 64 tiles before the first hit.
  auto ends = [&](int32_t kk) -> bool {
    if (kk >= total) return true;
    const uint64_t x = a.tile_info[kk];
    return !((x & kTileContinues) && (uint32_t)(x >> 32) == key);
  };
  int32_t kend = w + 1;
  const uint64_t near = __ballot(ends(w + 1 + lane));
  if (near) {
    kend = w + 1 + (int32_t)__builtin_ctzll(near);
  } else {
    const int32_t first = w + 1 + kWave;  // no tile before it ends
    for (int32_t lo = first;; lo += kWave * kWave) {
      const uint64_t coarse = __ballot(ends(lo + lane * kWave));
      if (!coarse) continue;
      // the first tile that ends lies in (lo + (j-1)*64, lo + j*64]
      const int j = __builtin_ctzll(coarse);
      int32_t base = lo + (j - 1) * kWave + 1;
      base = base > first ? base : first;
      kend = base + (int32_t)__builtin_ctzll(__ballot(ends(base + lane)));
      break;
    }
  }
  float g[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (own) {
#pragma unroll
    for (int i = 0; i < 4; ++i) g[i] = tail[i] + next[i];
  }
  if (cols) {
    // group 0 has added tile w + 1 already; past kend a load re-reads kk and
    // is not added
    for (int32_t kk = w + 1 + gi + (gi == 0 ? G : 0); kk <= kend; kk += kBatch * G) {
      f32x4 v8[kBatch];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) v8[j] = head(kk + j * G <= kend ? kk + j * G : kk);
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        if (kk + j * G <= kend) {
#pragma unroll
          for (int i = 0; i < 4; ++i) g[i] += v8[j][i];
        }
      }
    }
  }
  for (int q = 1; q < G; ++q) {
    float o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = __shfl(g[i], (lane % L) + q * L);
    if (gi == 0) {
#pragma unroll
      for (int i = 0; i < 4; ++i) g[i] += o[i];
    }
  }
  apply_update<TDT, 4>(m, a, (int64_t)(key - m.key_base), g, own, col, pre);
}

typedef void (*KernelFn)(BwdArgs);

template <int TDT>
KernelFn pick_tiles(int log2) {
  switch (log2) {
    case 0: return eb_bwd_tiles_kernel<TDT, 0>;
    case 1: return eb_bwd_tiles_kernel<TDT, 1>;
    case 2: return eb_bwd_tiles_kernel<TDT, 2>;
    case 3: return eb_bwd_tiles_kernel<TDT, 3>;
    case 4: return eb_bwd_tiles_kernel<TDT, 4>;
    case 5: return eb_bwd_tiles_kernel<TDT, 5>;
    case 6: return eb_bwd_tiles_kernel<TDT, 6>;
    default: return eb_bwd_tiles_kernel<TDT, -1>;
  }
}

// The workspace of eb_backward_update_noalloc: a static device array, one
// copy per GPU the library runs on, kept until the process ends.  Host code
// never uses its name as an address (on the host the name is only a
// stand-in); it uses the device address that hipGetSymbolAddress returns for
// the current device, looked up once per device.  No region of the
// workspace has to start at zero: each is written before it is read, so the
// contents a previous call left behind do not matter, but two calls that
// overlap on one GPU share the array and race.
constexpr size_t kScratchBytes = ::kScratchBytes;
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxScratchDevices];

// Device address of `scratch` on `device`, which must be the current device;
// nullptr if HIP cannot give it.
void *scratch_address(int device) {
  if (device < 0 || device >= kMaxScratchDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[device]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(::scratch)) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    g_scratch_ptr[device] = p;
  }
  return g_scratch_ptr[device];
}

// Workspace regions (each 256-byte aligned).
struct BwdLayout {
  size_t keys, skeys, spos, bag_of, tile_start, tile_info, carry, sort_tmp, total;
  size_t sort_bytes;
  int64_t tiles_ub;
  int32_t tile_size;
};

inline size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// Bits the largest sort key of handle h needs.
unsigned key_bits(const eb_tables *h) {
  const TableMeta &last = h->h_meta[h->num_tables - 1];
  const uint64_t max_key = (uint64_t)last.key_base + (uint64_t)last.num_rows;
  unsigned bits = 1;
  while (bits < 32 && (max_key >> bits) != 0) ++bits;
  return bits;
}

eb_status layout(const eb_tables *h, int64_t n, BwdLayout *L) {
  // Tiles of 64 positions keep short workloads spread over many wavefronts;
  // from about two million positions on, tiles of 128 carry fewer partial
  // sums (measured: 256 was slower at every size).
  int64_t chunks = n / (64 * 16384);
  chunks = chunks < 1 ? 1 : (chunks > 2 ? 2 : chunks);
  if (h->bwd_tile_chunks > 0) chunks = h->bwd_tile_chunks;
  L->tile_size = (int32_t)(64 * chunks);
  L->tiles_ub = (n + L->tile_size - 1) / L->tile_size + h->num_tables;
  size_t sort_bytes = 0;
  if (n > 0) {
    // scratch for either kind of value sorted with the keys (positions, or bag ids)
    size_t by_pos = 0, by_bag = 0;
    hipError_t e = rocprim::radix_sort_pairs<SortConfig>(nullptr, by_pos, static_cast<const uint32_t *>(nullptr),
                                             static_cast<uint32_t *>(nullptr), rocprim::counting_iterator<uint32_t>(0),
                                             static_cast<uint32_t *>(nullptr), (unsigned int)n, 0, key_bits(h),
                                             h->stream);
    if (e == hipSuccess)
      e = rocprim::radix_sort_pairs<SortConfig>(nullptr, by_bag, static_cast<const uint32_t *>(nullptr),
                                    static_cast<uint32_t *>(nullptr), static_cast<const uint32_t *>(nullptr),
                                    static_cast<uint32_t *>(nullptr), (unsigned int)n, 0, key_bits(h), h->stream);
    if (e != hipSuccess) return EB_ERR_HIP;
    sort_bytes = by_pos > by_bag ? by_pos : by_bag;
  }
  L->sort_bytes = sort_bytes;
  size_t off = 0;
  L->keys = off;
  off += align256(4 * (size_t)n);
  L->skeys = off;
  off += align256(4 * (size_t)n);
  L->spos = off;
  off += align256(4 * (size_t)n);
  L->bag_of = off;
  off += align256(4 * (size_t)n);
  L->tile_start = off;
  off += align256(4 * (size_t)(h->num_tables + 1));
  L->tile_info = off;
  off += align256(8 * (size_t)L->tiles_ub);
  L->carry = off;
  off += align256(4 * (size_t)2 * L->tiles_ub * h->max_dim);
  L->sort_tmp = off;
  off += align256(sort_bytes);
  L->total = off;
  return EB_OK;
}

}  // namespace
}  // namespace eb

using namespace eb;

extern "C" {

eb_status eb_backward_workspace_size(const eb_tables *h, int64_t num_indices, size_t *bytes) {
  if (!h || !bytes || num_indices < 0) return EB_ERR_INVALID_ARG;
  if (num_indices > INT32_MAX) return EB_ERR_UNSUPPORTED;
  BwdLayout L;
  const eb_status st = layout(h, num_indices, &L);
  if (st != EB_OK) return st;
  *bytes = L.total;
  return EB_OK;
}

}  // extern "C"

namespace eb {
namespace {

// The backward of eb_backward_update and eb_backward_update_noalloc, with
// its workspace given: the caller's, or (no_alloc) the library's static
// array, whose size is checked against what this call needs.
eb_status backward_update(const eb_tables *h, eb_tensor indices, eb_tensor offsets, eb_tensor per_sample_weights,
                          eb_pooling pooling, eb_tensor grad_out, int32_t optimizer, float learning_rate, float eps,
                          eb_tensor optimizer_state, void *workspace, size_t workspace_bytes, bool no_alloc) {
  if (!h) return EB_ERR_INVALID_ARG;
  if (!h->backward_ok) return EB_ERR_UNSUPPORTED;
  if (indices.elem_type != EB_I32 && indices.elem_type != EB_I64) return EB_ERR_DTYPE;
  if (offsets.elem_type != indices.elem_type) return EB_ERR_DTYPE;
  if (grad_out.elem_type != EB_T_F32) return EB_ERR_DTYPE;
  if (pooling != EB_POOL_SUM && pooling != EB_POOL_MEAN) return EB_ERR_INVALID_ARG;
  if (optimizer != EB_OPT_SGD && optimizer != EB_OPT_ROWWISE_ADAGRAD) return EB_ERR_INVALID_ARG;
  if (!offsets.data || !grad_out.data) return EB_ERR_INVALID_ARG;
  if (indices.numel < 0 || (indices.numel > 0 && !indices.data)) return EB_ERR_INVALID_ARG;
  if (indices.numel > INT32_MAX) return EB_ERR_UNSUPPORTED;
  const bool weighted = per_sample_weights.data != nullptr;
  if (weighted) {
    if (per_sample_weights.elem_type != EB_T_F32) return EB_ERR_DTYPE;
    if (pooling == EB_POOL_MEAN) return EB_ERR_INVALID_ARG;
    if (per_sample_weights.numel != indices.numel) return EB_ERR_SHAPE;
  }
  if (optimizer == EB_OPT_ROWWISE_ADAGRAD) {
    if (!optimizer_state.data) return EB_ERR_INVALID_ARG;
    if (optimizer_state.elem_type != EB_T_F32) return EB_ERR_DTYPE;
    if (optimizer_state.numel != h->total_rows) return EB_ERR_SHAPE;
  }
  if (offsets.numel < 2 || (offsets.numel - 1) % h->num_tables != 0) return EB_ERR_SHAPE;
  const int64_t num_bags = offsets.numel - 1;
  const int64_t batch = num_bags / h->num_tables;
  if (num_bags > INT32_MAX) return EB_ERR_SHAPE;
  if (grad_out.numel != batch * h->sum_dim) return EB_ERR_SHAPE;
  const size_t isz = indices.elem_type == EB_I64 ? 8 : 4;
  if (reinterpret_cast<uintptr_t>(grad_out.data) % 16 != 0 || reinterpret_cast<uintptr_t>(offsets.data) % isz != 0 ||
      reinterpret_cast<uintptr_t>(indices.data) % isz != 0 ||
      (weighted && reinterpret_cast<uintptr_t>(per_sample_weights.data) % 4 != 0) ||
      reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
    return EB_ERR_UNSUPPORTED;
  const int64_t n = indices.numel;
  BwdLayout L;
  eb_status st = layout(h, n, &L);
  if (st != EB_OK) return st;
  if (no_alloc && L.total > kScratchBytes) return EB_ERR_UNSUPPORTED;  // past the static array
  if (n == 0) return EB_OK;  // no row was read: nothing to update

  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return EB_ERR_HIP;
  if (cur != h->device && hipSetDevice(h->device) != hipSuccess) return EB_ERR_HIP;
  if (no_alloc) {
    // the static array's address on the handle's device (now current)
    workspace = scratch_address(h->device);
    workspace_bytes = kScratchBytes;
    if (!workspace) {
      if (cur != h->device) (void)hipSetDevice(cur);
      return EB_ERR_HIP;
    }
  }
  if (!workspace || workspace_bytes < L.total) {
    if (cur != h->device) (void)hipSetDevice(cur);
    return EB_ERR_INVALID_ARG;
  }

  unsigned char *ws = static_cast<unsigned char *>(workspace);
  BwdArgs a;
  a.meta = h->d_meta;
  a.ctx.err = h->d_err;
  a.ctx.zero = h->d_zero;
  a.ctx.one = 1.0f;
  a.indices = indices.data;
  a.offsets = offsets.data;
  a.weights = static_cast<const float *>(per_sample_weights.data);
  a.grad = static_cast<const float *>(grad_out.data);
  a.state = static_cast<float *>(const_cast<void *>(optimizer_state.data));
  a.keys = reinterpret_cast<uint32_t *>(ws + L.keys);
  a.bag_of = reinterpret_cast<int32_t *>(ws + L.bag_of);
  a.skeys = reinterpret_cast<const uint32_t *>(ws + L.skeys);
  a.spos = reinterpret_cast<const uint32_t *>(ws + L.spos);
  a.tile_start = reinterpret_cast<int32_t *>(ws + L.tile_start);
  a.tile_info = reinterpret_cast<uint64_t *>(ws + L.tile_info);
  a.carry = reinterpret_cast<float *>(ws + L.carry);
  a.num_indices = n;
  a.grad_ld = h->sum_dim;
  a.num_bags = (int32_t)num_bags;
  a.batch = (int32_t)batch;
  a.num_tables = h->num_tables;
  a.idx64 = indices.elem_type == EB_I64;
  a.coef = pooling == EB_POOL_MEAN ? 2 : (weighted ? 1 : 0);
  a.sorted_bags = weighted ? 0 : 1;
  a.opt = optimizer;
  a.lr = learning_rate;
  a.eps = eps;
  a.tile_size = L.tile_size;
  a.max_dim = h->max_dim;
  a.xcd_remap = h->bwd_xcd_remap;
  int64_t k = 1;
  {
    const int64_t per_slot = num_bags / kResidentWaves;
    while ((k + 1) * (k + 1) <= per_slot) ++k;
    k = k > kMaxBagsPerWave ? kMaxBagsPerWave : k;
  }
  a.bags_per_wave = (int32_t)k;
  a.groups_per_table = (int32_t)((batch + k - 1) / k);
  a.num_waves = (int32_t)((int64_t)a.groups_per_table * h->num_tables);

  hipError_t e = hipSuccess;
  if (h->checked) e = hipMemsetAsync(h->d_err, 0, sizeof(int), h->stream);
  // 1. keys
  if (e == hipSuccess) {
    const unsigned grid = (unsigned)((a.num_waves + kWavesPerBlock - 1) / kWavesPerBlock);
    hipLaunchKernelGGL(eb_bwd_keys_kernel, dim3(grid), dim3(kBlock), 0, h->stream, a);
    e = hipGetLastError();
  }
  // 2. sort (key, bag id) pairs, or (key, position) pairs when the weights
  //    (per position) are needed, on the bits the largest key needs
  if (e == hipSuccess) {
    const unsigned end_bit = key_bits(h);
    size_t tmp = L.sort_bytes;
    if (a.sorted_bags)
      e = rocprim::radix_sort_pairs<SortConfig>(ws + L.sort_tmp, tmp, a.keys, const_cast<uint32_t *>(a.skeys),
                                    reinterpret_cast<const uint32_t *>(a.bag_of), const_cast<uint32_t *>(a.spos),
                                    (unsigned int)n, 0, end_bit, h->stream);
    else
      e = rocprim::radix_sort_pairs<SortConfig>(ws + L.sort_tmp, tmp, a.keys, const_cast<uint32_t *>(a.skeys),
                                    rocprim::counting_iterator<uint32_t>(0), const_cast<uint32_t *>(a.spos),
                                    (unsigned int)n, 0, end_bit, h->stream);
  }
  // 3. tiles: pool and update (the first tile of each table came with the keys)
  const unsigned tgrid = (unsigned)((L.tiles_ub + kTileWaves - 1) / kTileWaves);
  const unsigned fgrid = (unsigned)((L.tiles_ub + kWavesPerBlock - 1) / kWavesPerBlock);
  // one launch per storage type present; fixed row width when all tables share it
  int32_t glog2 = log2_lanes_per_row(4 * h->h_meta[0].dim);
  for (int32_t t = 1; t < h->num_tables; ++t)
    if (log2_lanes_per_row(4 * h->h_meta[t].dim) != glog2) glog2 = -1;
  for (int dt = 0; dt < 2 && e == hipSuccess; ++dt) {
    if (!(h->dtype_mask & (1 << dt))) continue;
    hipLaunchKernelGGL(dt == kF32 ? pick_tiles<kF32>(glog2) : pick_tiles<kF16>(glog2), dim3(tgrid),
                       dim3(kWave * kTileWaves), 0,
                       h->stream, a);
    e = hipGetLastError();
  }
  // 4. runs that cross tiles
  for (int dt = 0; dt < 2 && e == hipSuccess; ++dt) {
    if (!(h->dtype_mask & (1 << dt))) continue;
    hipLaunchKernelGGL(dt == kF32 ? eb_bwd_fixup_kernel<kF32> : eb_bwd_fixup_kernel<kF16>, dim3(fgrid), dim3(kBlock),
                       0, h->stream, a);
    e = hipGetLastError();
  }
  if (e == hipSuccess && h->checked) {
    int herr = 0;
    e = hipMemcpyAsync(&herr, h->d_err, sizeof(int), hipMemcpyDeviceToHost, h->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h->stream);
    if (e == hipSuccess && (herr & kErrOffsets)) st = EB_ERR_OFFSETS;
    else if (e == hipSuccess && (herr & kErrIndex)) st = EB_ERR_INDEX_OOB;
  }
  if (e != hipSuccess) st = EB_ERR_HIP;
  if (cur != h->device) (void)hipSetDevice(cur);
  return st;
}

}  // namespace
}  // namespace eb

extern "C" {

eb_status eb_backward_update(const eb_tables *h, eb_tensor indices, eb_tensor offsets, eb_tensor per_sample_weights,
                             eb_pooling pooling, eb_tensor grad_out, int32_t optimizer, float learning_rate,
                             float eps, eb_tensor optimizer_state, void *workspace, size_t workspace_bytes) {
  return backward_update(h, indices, offsets, per_sample_weights, pooling, grad_out, optimizer, learning_rate, eps,
                         optimizer_state, workspace, workspace_bytes, false);
}

eb_status eb_backward_update_noalloc(const eb_tables *h, eb_tensor indices, eb_tensor offsets,
                                     eb_tensor per_sample_weights, eb_pooling pooling, eb_tensor grad_out,
                                     int32_t optimizer, float learning_rate, float eps, eb_tensor optimizer_state) {
  return backward_update(h, indices, offsets, per_sample_weights, pooling, grad_out, optimizer, learning_rate, eps,
                         optimizer_state, nullptr, 0, true);
}

}  // extern "C"
