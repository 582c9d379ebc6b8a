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
//   1. every position gets a sort element (its row, or the table's sentinel
//      row, above its table-local bag id or its position), and each table's
//      first tile and sort blocks are found from the offsets;
//   2. each table's elements are radix-sorted by row, least significant digit
//      first, one stable pass per digit: each row's occurrences become one
//      run, in position order, and each table's positions stay inside that
//      table's range of the sorted array;
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

#include <atomic>
#include <mutex>

#include "eb_device.h"

// The static workspace of eb_backward_update_noalloc (see scratch_address).
constexpr size_t kScratchBytes = (size_t)EB_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace eb {
namespace {

constexpr uint32_t kNoKey = 0xFFFFFFFFu;  // larger than any key (keys fit below it)
constexpr uint8_t kTileContinues = 1;      // the tile's last run goes on into the next tile
constexpr uint8_t kTileOwnsRun = 2;        // ... and started in this tile: this tile finishes it
constexpr int kOptRowwiseAdagrad = 1;

// The sort (step 2): workgroups of 512 threads, digits of up to 9 bits (one
// digit per thread where a workgroup handles all digits), up to 4 passes
// (rows of up to 32 bits).
constexpr int kSortThreads = 512;
constexpr int kSortWaves = kSortThreads / kWave;
constexpr int kSortRadixMax = 512;
constexpr int kSortMaxPasses = 4;

struct BwdArgs {
  const TableMeta *meta;
  GatherCtx ctx;
  const void *indices;
  const void *offsets;
  const float *weights;
  const float *grad;      // grad_out [B, sum D]
  float *state;           // row-wise Adagrad state [sum R]
  int32_t *bag_of;        // [N] bag id by position (positions sorted: weighted pooling)
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
  // the sort (step 2)
  void *elems[2];         // [N] sort elements: elems[0] by position, then alternating per pass
  int4 *sblocks;          // [sort blocks] {table, first position, end position, table's first position}
  int32_t *sort_nblocks;  // number of sort blocks
  uint32_t *hist;         // [T][passes][radix] digit counts per table
  uint64_t *status;       // [passes][sort blocks][radix] per-block digit counts for the look-back
  uint4 *zero;            // hist and status: cleared by the keys kernel
  int64_t zero_words;     // 16-byte words from `zero`
  int32_t sort_block;     // positions per sort block
  int32_t sort_nblk_ub;   // sort blocks the launch provides for
  int32_t sort_passes;
  int32_t sort_bits;      // digit bits per pass
  int32_t sort_wide;      // 64-bit elements: row << 32 | value; else row << vshift | value
  int32_t sort_vshift;
  uint32_t sort_vmask;
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

// Exclusive scan of one int64 per thread over a workgroup of NT threads
// (part: 2 * NT / 64 slots of LDS); total receives the sum of all.
template <int NT>
__device__ __forceinline__ int64_t block_exclusive_scan(int64_t x, int64_t *part, int64_t &total) {
  constexpr int kWaves = NT / kWave;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1), wave = tid / kWave;
  int64_t incl = x;
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
  total = part[2 * kWaves - 1];
  const int64_t r = incl - x + (wave > 0 ? part[kWaves + wave - 1] : 0);
  __syncthreads();  // part may be reused
  return r;
}

// Step 3a: first tile of every table, an exclusive scan of the tables' tile
// counts, and the sort blocks of step 2 (each table's positions cut into
// pieces of sort_block), by one workgroup of NT threads.  Both depend on the
// offsets alone, so the keys kernel's first workgroup does this before its own
// positions.
template <int NT>
__device__ __forceinline__ void scan_tables(const BwdArgs &a, int64_t *part) {
  const int T = a.num_tables;
  const int tid = threadIdx.x;
  const int per = (T + NT - 1) / NT;
  const int t0 = tid * per < T ? tid * per : T;
  const int t1 = t0 + per < T ? t0 + per : T;
  const int64_t SB = a.sort_block;
  int64_t tiles = 0, blocks = 0;
  for (int t = t0; t < t1; ++t) {
    int64_t p0, p1;
    table_range(a, t, p0, p1);
    tiles += (p1 - p0 + a.tile_size - 1) / a.tile_size;
    blocks += (p1 - p0 + SB - 1) / SB;
  }
  int64_t total_tiles, total_blocks;
  int64_t tile = block_exclusive_scan<NT>(tiles, part, total_tiles);
  int64_t blk = block_exclusive_scan<NT>(blocks, part, total_blocks);
  if (tid == 0) {
    a.tile_start[T] = (int32_t)total_tiles;
    *a.sort_nblocks = (int32_t)total_blocks;
  }
  for (int t = t0; t < t1; ++t) {
    a.tile_start[t] = (int32_t)tile;
    int64_t p0, p1;
    table_range(a, t, p0, p1);
    tile += (p1 - p0 + a.tile_size - 1) / a.tile_size;
    for (int64_t s = p0; s < p1; s += SB, ++blk)
      a.sblocks[blk] = make_int4(t, (int32_t)s, (int32_t)(s + SB < p1 ? s + SB : p1), (int32_t)p0);
  }
}

// Sort elements (and, for weighted pooling, bag ids) of positions [P0, P1)
// (bags g0 .. g0 + nb - 1 of table t, whose offsets lane j holds in my_off).
// kKeyChunks chunks of 64 positions per round: every index load of a round is
// issued before its first element is stored, and none sits behind a branch (a
// position past P1 re-reads P1 - 1), so a round costs one memory round trip.
// Returns whether this lane saw an index outside the table.
template <typename IT>
__device__ __forceinline__ bool key_positions(const BwdArgs &a, const TableMeta &m, int64_t P0, int64_t P1,
                                              int64_t my_off, int nb, int32_t g0, int32_t b0) {
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
    // bag of each position: the number of the run's later bags that start
    // at or before it (each bag's offset read once for the four chunks)
    int jv[kKeyChunks];
#pragma unroll
    for (int u = 0; u < kKeyChunks; ++u) jv[u] = 0;
    for (int jj = 1; jj < nb; ++jj) {
      const int64_t o = readlane64(my_off, jj);
#pragma unroll
      for (int u = 0; u < kKeyChunks; ++u) jv[u] += o <= c + u * kWave + lane ? 1 : 0;
    }
#pragma unroll
    for (int u = 0; u < kKeyChunks; ++u) {
      const int64_t p = c + u * kWave + lane;
      if (p < P1) {
        const int j = jv[u];
        const bool ok = r[u] >= 0 && r[u] < m.num_rows;
        oob |= !ok;
        const uint32_t row = ok ? (uint32_t)r[u] : (uint32_t)m.num_rows;
        // unweighted pooling carries the table-local bag id; weighted pooling
        // the position, whose weight and bag the tiles kernel looks up
        const uint32_t v = a.sorted_bags ? (uint32_t)(b0 + j) : (uint32_t)p;
        if (a.sort_wide) static_cast<uint64_t *>(a.elems[0])[p] = ((uint64_t)row << 32) | v;
        else static_cast<uint32_t *>(a.elems[0])[p] = (row << a.sort_vshift) | v;
        if (!a.sorted_bags) a.bag_of[p] = g0 + j;
      }
    }
  }
  return oob;
}

// Step 1: sort element of every position.  A wavefront takes a run of
// consecutive bags of one table and walks their positions 64 at a time (the
// same work map as the forward).  An index outside its table gets the table's
// sentinel row (one past its last row), which sorts after the table's rows
// and is skipped later.  The kernel also clears the sort's counters.
__global__ __launch_bounds__(kBlock) void eb_bwd_keys_kernel(BwdArgs a) {
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < a.zero_words; i += (int64_t)gridDim.x * kBlock)
    a.zero[i] = make_uint4(0u, 0u, 0u, 0u);
  if (blockIdx.x == 0) {
    // every thread of the workgroup, before any wavefront can leave
    __shared__ int64_t part[2 * kWavesPerBlock];
    scan_tables<kBlock>(a, part);
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
  const bool oob = a.idx64 ? key_positions<int64_t>(a, m, P0, P1, my_off, nb, g0, b0)
                           : key_positions<int32_t>(a, m, P0, P1, my_off, nb, g0, b0);
  if (__ballot(oob)) {
    if (lane == 0) atomicOr(a.ctx.err, kErrIndex);
  }
}

// Step 2: the sort.  Each table's elements are sorted by row, least
// significant digit first; a pass is a stable partition by one digit of the
// row inside every table's range of positions, which is cut into sort blocks
// of sort_block positions.  The digit counts of every table and pass come
// first (eb_bwd_sort_hist_kernel).  In a pass (eb_bwd_sort_pass_kernel) a
// workgroup ranks a sort block's elements by digit in LDS, and finds where its
// digits go from the blocks before it in the same table: it publishes its own
// digit counts, then walks back over its predecessors' published counts until
// one of them holds the sum over every block before it, and publishes that sum
// with its own counts added.  This is the decoupled look-back of single-pass
// prefix scans (Merrill and Garland, 2016), as radix sorts with one pass per
// digit use it.  Workgroup b sorts block b, and a block waits only for
// earlier blocks of its table.  The workgroups of one launch start in order
// on each XCD, so when block u is the lowest unfinished one, every workgroup
// ahead of it on its XCD has finished: u is running or can start, and it
// waits for nothing unfinished.  So no block waits for one that cannot run,
// however many of the launch's workgroups the GPU holds at once.  (A ticket
// counter that orders workgroups as they start costs every workgroup an
// atomic on one address, which serialised: about 37 ns each.)  Every wait is
// bounded besides, so that a wait that never ended would raise kErrSortWait
// and let the workgroup go on rather than hang.
constexpr int kHistThreads = 512;
constexpr uint32_t kLbAggregate = 1;    // status word: the block's own counts
constexpr uint32_t kLbPrefix = 2;       // ... counts of every block of the table up to and including it
constexpr int kSortSpinLimit = 1 << 18;
constexpr int kLookBack = 8;  // predecessors read per look-back round trip

// row of a sort element
template <typename E>
__device__ __forceinline__ uint32_t elem_row(const BwdArgs &a, E e) {
  if constexpr (sizeof(E) == 8) return (uint32_t)(e >> 32);
  else return e >> a.sort_vshift;
}

// Digit counts of each table for every pass, from the elements in position
// order: one workgroup per sort block counts in LDS, with all of the block's
// loads in flight at once, and adds its counts to the table's (integer
// additions: the totals do not depend on their order).
template <typename E>
__global__ __launch_bounds__(kHistThreads) void eb_bwd_sort_hist_kernel(BwdArgs a) {
  constexpr int U = 16;  // a block's elements per thread
  __shared__ uint32_t h[kSortMaxPasses * kSortRadixMax];
  const int tid = threadIdx.x;
  const int np = a.sort_passes, bits = a.sort_bits, radix = 1 << bits;
  const uint32_t dmask = (uint32_t)radix - 1u;
  const int nh = np * radix;
  for (int i = tid; i < nh; i += kHistThreads) h[i] = 0u;
  const int32_t b = blockIdx.x;
  if (b >= *a.sort_nblocks) return;
  const int4 sb = a.sblocks[b];
  const E *src = static_cast<const E *>(a.elems[0]);
  __syncthreads();
  for (int32_t p = sb.y + tid; p < sb.z; p += U * kHistThreads) {
    E e[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int32_t q = p + u * kHistThreads;
      e[u] = src[q < sb.z ? q : p];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (p + u * kHistThreads < sb.z) {
        const uint32_t row = elem_row<E>(a, e[u]);
        const uint64_t below = (1ull << (threadIdx.x & (kWave - 1))) - 1ull;
        for (int q = 0; q + 1 < np; ++q) atomicAdd(&h[q * radix + ((row >> (q * bits)) & dmask)], 1u);
        // the top digit: the lanes that share the first active lane's (often
        // most of them: a small table's rows, a power-law's low rows) add
        // once together; lanes that add to one LDS word in one instruction
        // take turns
        const int q = np - 1;
        const uint32_t d = (row >> (q * bits)) & dmask;
        const uint32_t d0 = __builtin_amdgcn_readfirstlane(d);
        const uint64_t same = __ballot(d == d0);
        if (d != d0) atomicAdd(&h[q * radix + d], 1u);
        else if ((same & below) == 0) atomicAdd(&h[q * radix + d0], (uint32_t)__builtin_popcountll(same));
      }
    }
  }
  __syncthreads();
  uint32_t *g = a.hist + (size_t)sb.x * nh;
  for (int i = tid; i < nh; i += kHistThreads) {
    const uint32_t v = h[i];
    if (v) atomicAdd(g + i, v);
  }
}

// Sort block b of a pass (the body of eb_bwd_sort_pass_kernel's loop).
template <typename E, int IPT>
__device__ __forceinline__ void sort_block(const BwdArgs &a, int32_t pass, int32_t b, E *stage,
                                           uint32_t (*cnt)[kSortRadixMax], int32_t *loff, int32_t *goff,
                                           int64_t *part, int tid, int lane, int w) {
  __syncthreads();  // the previous block's reads of LDS are done
  for (int i = tid; i < kSortWaves * kSortRadixMax; i += kSortThreads) (&cnt[0][0])[i] = 0;
  __syncthreads();
  const int4 sb = a.sblocks[b];  // {table, start, end, table's first position}
  const int bits = a.sort_bits, radix = 1 << bits;
  const uint32_t dmask = (uint32_t)radix - 1u;
  const int shift = (sizeof(E) == 8 ? 32 : a.sort_vshift) + pass * bits;
  const E *src = static_cast<const E *>(a.elems[pass & 1]);
  const int32_t n = sb.z - sb.y;

  // elements past the block's end get the largest digit: they rank after
  // every element of the block and are not stored
  E e[IPT];
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const int k = w * kWave * IPT + i * kWave + lane;
    e[i] = k < n ? src[sb.y + k] : ~(E)0;
  }
  const uint32_t tcount =
      tid < radix ? a.hist[((size_t)sb.x * a.sort_passes + pass) * radix + tid] : 0u;
  // stable rank within the wave: the lanes holding the same digit are found
  // with one ballot per digit bit; the lowest of them adds the group to the
  // wave's count of that digit (an LDS add that returns the count before it:
  // one wave's LDS operations take effect in order, so the items' adds need
  // not wait for each other) and the others read that count from it
  // (four items at a time, which bounds the registers the adds in flight hold)
  uint32_t dg[IPT], rk[IPT];
  const uint64_t below_me = (1ull << lane) - 1ull;
#pragma unroll
  for (int i0 = 0; i0 < IPT; i0 += 4) {
    uint32_t lead[4], old[4], plo[4], phi[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      dg[i0 + u] = (uint32_t)(e[i0 + u] >> shift) & dmask;
      plo[u] = ~0u;
      phi[u] = ~0u;
    }
    // a lane keeps the lanes whose bit q equals its own: the ballot of bit
    // q, complemented where the lane's bit is 0 (m: the bit copied into
    // every bit of a word, one signed bit-field extract).  Bit by bit for
    // the four items at once, so their four chains of dependent operations
    // interleave.
    for (int q = 0; q < bits; ++q) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint32_t m = (uint32_t)__builtin_amdgcn_sbfe((int)dg[i0 + u], (uint32_t)q, 1u);
        const uint64_t bal = __ballot(m != 0u);
        // p & ~(ballot ^ m) as one three-input bitwise operation per half
        // (truth table 0x90: inputs p, ballot, m)
        plo[u] = __builtin_amdgcn_bitop3_b32(plo[u], (uint32_t)bal, m, 0x90);
        phi[u] = __builtin_amdgcn_bitop3_b32(phi[u], (uint32_t)(bal >> 32), m, 0x90);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u;
      const uint64_t peers = ((uint64_t)phi[u] << 32) | plo[u];
      const uint64_t below = peers & below_me;
      rk[i] = (uint32_t)__builtin_popcountll(below);
      lead[u] = (uint32_t)__builtin_ctzll(peers);
      old[u] = below == 0 ? atomicAdd(&cnt[w][dg[i]], (uint32_t)__builtin_popcountll(peers)) : 0u;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) rk[i0 + u] += (uint32_t)__shfl((int)old[u], (int)lead[u]);
  }
  __syncthreads();
  // per digit: counts of the earlier waves, and the block's count, published
  // at once for the blocks after this one
  const bool first = sb.y == sb.w;
  uint64_t *status = a.status + (size_t)pass * a.sort_nblk_ub * radix;
  uint32_t bcount = 0;
  if (tid < radix) {
    uint32_t run = 0;
#pragma unroll
    for (int ww = 0; ww < kSortWaves; ++ww) {
      const uint32_t c = cnt[ww][tid];
      cnt[ww][tid] = run;
      run += c;
    }
    bcount = run;
    __hip_atomic_store(status + (size_t)b * radix + tid, ((uint64_t)(first ? kLbPrefix : kLbAggregate) << 32) | bcount,
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  // exclusive scans over the digits: the block's local slots, and where each
  // digit starts in the table
  // (one scan of both: the block's counts sum to at most SB, so they stay in
  // the low 32 bits)
  int64_t total;
  const int64_t both =
      block_exclusive_scan<kSortThreads>(((int64_t)tcount << 32) | (int64_t)bcount, part, total);
  const int32_t lo = (int32_t)(both & 0xFFFFFFFF);
  const int32_t tb = (int32_t)(both >> 32);
  const int32_t table_end = sb.w + (int32_t)(total >> 32);  // the table's element count is its digits' total
  if (tid < radix) loff[tid] = lo;
  __syncthreads();
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const uint32_t slot = (uint32_t)loff[dg[i]] + cnt[w][dg[i]] + rk[i];
    if (slot < (uint32_t)(kSortThreads * IPT)) stage[slot] = e[i];  // always: the ranks are a permutation of the block
  }
  // look-back: the digit's count over the table's blocks before this one,
  // kLookBack predecessors' status words per round trip, nearest first; the
  // table's first block (jmin) holds a prefix, so the walk stops there
  if (tid < radix) {
    uint32_t before = 0;
    if (!first) {
      const int32_t jmin = b - (sb.y - sb.w) / a.sort_block;
      int32_t j = b - 1;
      for (bool done = false; !done;) {
        uint64_t x[kLookBack];
#pragma unroll
        for (int u = 0; u < kLookBack; ++u) {
          const int32_t jj = j - u > jmin ? j - u : jmin;
          x[u] = __hip_atomic_load(status + (size_t)jj * radix + tid, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        int ready = kLookBack;  // the nearest predecessor not yet published
#pragma unroll
        for (int u = 0; u < kLookBack; ++u) {
          if (!done && ready == kLookBack) {
            if ((x[u] >> 32) == 0) {
              ready = u;
            } else {
              before += (uint32_t)x[u];
              done = (x[u] >> 32) == kLbPrefix;
            }
          }
        }
        if (done) break;
        j -= ready;
        if (ready < kLookBack) {
          // wait for block j (bounded), then read on from it
          const uint64_t *sj = status + (size_t)j * radix + tid;
          uint64_t y = __hip_atomic_load(sj, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          for (int spin = 0; (y >> 32) == 0 && spin < kSortSpinLimit; ++spin) {
            __builtin_amdgcn_s_sleep(1);
            y = __hip_atomic_load(sj, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          }
          if ((y >> 32) == 0) {
            atomicOr(a.ctx.err, kErrSortWait);
            break;
          }
        }
      }
      __hip_atomic_store(status + (size_t)b * radix + tid, ((uint64_t)kLbPrefix << 32) | (before + bcount),
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    goff[tid] = sb.w + tb + (int32_t)before - lo;
  }
  __syncthreads();
  // store in local order: consecutive slots of one digit go to consecutive
  // positions
  const bool last = pass == a.sort_passes - 1;
  E *dst = static_cast<E *>(a.elems[(pass + 1) & 1]);
  uint32_t key_base = 0, rows = 0, bag_base = 0;
  if (last) {
    key_base = a.meta[sb.x].key_base;
    rows = (uint32_t)a.meta[sb.x].num_rows;
    bag_base = (uint32_t)sb.x * (uint32_t)a.batch;
  }
#pragma unroll 4
  for (int i = 0; i < IPT; ++i) {
    const int k = i * kSortThreads + tid;
    if (k < n) {
      const E x = stage[k];
      const int32_t out = goff[(uint32_t)(x >> shift) & dmask] + k;
      if (out < sb.w || out >= table_end) continue;  // never: counts and ranks agree
      if (!last) {
        dst[out] = x;
      } else {
        // the row (the sentinel for an index outside the table) and the bag
        // id or position; a value out of range, which only positions the
        // keys kernel never wrote (broken offsets) can hold, gets the
        // sentinel row, which later steps skip
        uint32_t row = elem_row<E>(a, x);
        uint32_t v = (uint32_t)x & a.sort_vmask;
        const bool bad = a.sorted_bags ? v >= (uint32_t)a.batch : (int64_t)v >= a.num_indices;
        if (row > rows || bad) {
          row = rows;
          v = 0;
        }
        const_cast<uint32_t *>(a.skeys)[out] = key_base + row;
        const_cast<uint32_t *>(a.spos)[out] = a.sorted_bags ? bag_base + v : v;
      }
    }
  }
}

// One pass: sort block blockIdx.x (and, were the grid smaller than the
// blocks, blockIdx.x + gridDim.x, ...), partitioned by digit `pass` of the row.  Element k of a block (position start + k) is item
// k / 64 % IPT of wave k / (64 * IPT), lane k % 64; the block's stable order
// is k.
template <typename E, int IPT>
// (12 elements per thread: held to 128 VGPRs, 4 waves per SIMD, so that two
// workgroups share a compute unit; the compiler's own choice was 135, one.)
__global__ __launch_bounds__(kSortThreads) __attribute__((amdgpu_waves_per_eu(IPT == 12 ? 4 : 1, 8)))
void eb_bwd_sort_pass_kernel(BwdArgs a, int32_t pass) {
  constexpr int SB = kSortThreads * IPT;
  __shared__ E stage[SB];
  __shared__ uint32_t cnt[kSortWaves][kSortRadixMax];  // per wave: digit counts, then counts of earlier waves
  __shared__ int32_t loff[kSortRadixMax];               // first local slot of each digit
  __shared__ int32_t goff[kSortRadixMax];               // output position of a digit's local slot 0
  __shared__ int64_t part[2 * kSortWaves];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
  const int32_t nblk = *a.sort_nblocks;
  for (int32_t b = blockIdx.x; b < nblk; b += gridDim.x) {
    sort_block<E, IPT>(a, pass, b, stage, cnt, loff, goff, part, tid, lane, w);
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

// Elements per thread of the sort's pass kernels, and the kernels (32-bit
// elements, then 64-bit, each by kSortItems).
constexpr int kSortItems[4] = {4, 8, 12, 16};
void (*const kSortPass[8])(BwdArgs, int32_t) = {
    eb_bwd_sort_pass_kernel<uint32_t, 4>,  eb_bwd_sort_pass_kernel<uint32_t, 8>,
    eb_bwd_sort_pass_kernel<uint32_t, 12>, eb_bwd_sort_pass_kernel<uint32_t, 16>,
    eb_bwd_sort_pass_kernel<uint64_t, 4>,  eb_bwd_sort_pass_kernel<uint64_t, 8>,
    eb_bwd_sort_pass_kernel<uint64_t, 12>, eb_bwd_sort_pass_kernel<uint64_t, 16>};

// Workgroups of sort pass kernel `which` that device `device` holds at once
// (its compute units times the kernel's occupancy per unit), and its compute
// units; looked up once per device and kernel.
std::atomic<int64_t> g_resident[kMaxScratchDevices][8];
std::atomic<int32_t> g_cus[kMaxScratchDevices];

hipError_t resident_grid(int device, int which, int64_t *grid, int32_t *cus) {
  if (device < 0 || device >= kMaxScratchDevices) return hipErrorInvalidDevice;
  int64_t g = g_resident[device][which].load(std::memory_order_relaxed);
  int32_t c = g_cus[device].load(std::memory_order_relaxed);
  if (g <= 0 || c <= 0) {
    int n = 0, per_cu = 0;
    hipError_t e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, device);
    if (e == hipSuccess)
      e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void *>(kSortPass[which]),
                                                       kSortThreads, 0);
    if (e != hipSuccess) return e;
    c = n > 0 ? n : 1;
    g = (int64_t)c * (per_cu > 0 ? per_cu : 1);
    g_resident[device][which].store(g, std::memory_order_relaxed);
    g_cus[device].store(c, std::memory_order_relaxed);
  }
  *grid = g;
  *cus = c;
  return hipSuccess;
}

// Elements per thread of this call's sort (kernel `which`, sort blocks of
// 512 * items positions, one workgroup per block): the fewest rounds of
// resident workgroups over the blocks; among those, the largest blocks that
// still give every compute unit one (fewer blocks shorten the look-back and
// cost less per block, but a block per unit keeps the GPU busy).
hipError_t choose_sort_items(const eb_tables *h, int64_t n, bool wide, int *which, int64_t *nblk_ub,
                             int64_t *grid) {
  int64_t best_rounds = -1;
  for (int c = 0; c < 4; ++c) {
    if (h->bwd_sort_items > 0 && kSortItems[c] != h->bwd_sort_items) continue;
    const int k = (wide ? 4 : 0) + c;
    const int64_t sb = (int64_t)kSortThreads * kSortItems[c];
    const int64_t blocks = (n + sb - 1) / sb + h->num_tables;
    int64_t g = 0;
    int32_t cus = 0;
    const hipError_t e = resident_grid(h->device, k, &g, &cus);
    if (e != hipSuccess) return e;
    const int64_t rounds = (blocks + g - 1) / g;
    if (best_rounds < 0 || rounds < best_rounds || (rounds == best_rounds && blocks >= cus)) {
      best_rounds = rounds;
      *which = k;
      *nblk_ub = blocks;
      *grid = blocks;
    }
  }
  return best_rounds < 0 ? hipErrorInvalidValue : hipSuccess;
}

// Workspace regions (each 256-byte aligned).
struct BwdLayout {
  size_t elems[2], bag_of, tile_start, tile_info, carry, sblocks, nblocks, zero, total;
  size_t hist_bytes;  // the digit counts at `zero`; the look-back status follows
  int64_t tiles_ub;
  int32_t tile_size;
  // the sort
  int32_t row_bits, passes, bits;
  int64_t nblk_max;
};

inline size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// Bits of x (0 for 0).
unsigned bit_width(uint64_t x) {
  unsigned b = 0;
  while (b < 64 && (x >> b) != 0) ++b;
  return b;
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
  // The sort: rows up to the largest table's sentinel (its row count), in as
  // few passes of at most 9 bits as cover them, split evenly.
  int64_t max_rows = 0;
  for (int32_t t = 0; t < h->num_tables; ++t)
    max_rows = h->h_meta[t].num_rows > max_rows ? h->h_meta[t].num_rows : max_rows;
  L->row_bits = (int32_t)bit_width((uint64_t)max_rows);
  if (L->row_bits < 1) L->row_bits = 1;
  L->passes = (L->row_bits + 8) / 9;
  L->bits = (L->row_bits + L->passes - 1) / L->passes;
  // sized for the smallest sort block (the most blocks); a call uses a part
  L->nblk_max = (n + kSortThreads * kSortItems[0] - 1) / (kSortThreads * kSortItems[0]) + h->num_tables;
  const size_t radix = (size_t)1 << L->bits;
  size_t off = 0;
  for (int i = 0; i < 2; ++i) {  // 8 bytes per element: 64-bit elements, or the sorted keys and values
    L->elems[i] = off;
    off += align256(8 * (size_t)n);
  }
  L->bag_of = off;
  off += align256(4 * (size_t)n);
  L->tile_start = off;
  off += align256(4 * (size_t)(h->num_tables + 1));
  L->tile_info = off;
  off += align256(8 * (size_t)L->tiles_ub);
  L->carry = off;
  off += align256(4 * (size_t)2 * L->tiles_ub * h->max_dim);
  L->sblocks = off;
  off += align256(16 * (size_t)L->nblk_max);
  L->nblocks = off;
  off += 256;
  // cleared by the keys kernel: digit counts, look-back status
  L->zero = off;
  L->hist_bytes = align256(4 * (size_t)h->num_tables * L->passes * radix);
  off += L->hist_bytes + align256(8 * (size_t)L->passes * L->nblk_max * radix);
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
  a.bag_of = reinterpret_cast<int32_t *>(ws + L.bag_of);
  // pass q reads elems[q % 2] and writes elems[(q + 1) % 2]; the last pass
  // writes the sorted keys and values into the buffer it does not read
  a.elems[0] = ws + L.elems[0];
  a.elems[1] = ws + L.elems[1];
  a.skeys = reinterpret_cast<const uint32_t *>(ws + L.elems[L.passes % 2]);
  a.spos = a.skeys + n;
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
  a.sblocks = reinterpret_cast<int4 *>(ws + L.sblocks);
  a.sort_nblocks = reinterpret_cast<int32_t *>(ws + L.nblocks);
  a.zero = reinterpret_cast<uint4 *>(ws + L.zero);
  a.hist = reinterpret_cast<uint32_t *>(ws + L.zero);
  a.status = reinterpret_cast<uint64_t *>(ws + L.zero + L.hist_bytes);
  a.sort_passes = L.passes;
  a.sort_bits = L.bits;
  {
    // an element holds the row above the value (table-local bag id, or
    // position): in 32 bits when both fit
    const int32_t vbits = (int32_t)bit_width(weighted ? (uint64_t)(n - 1) : (uint64_t)(batch - 1));
    a.sort_wide = L.row_bits + vbits > 32 ? 1 : 0;
    a.sort_vshift = a.sort_wide ? 32 : vbits;
    a.sort_vmask = a.sort_wide ? 0xFFFFFFFFu : (uint32_t)(((uint64_t)1 << vbits) - 1);
  }
  int sort_kernel = 0;
  int64_t sort_nblk = 0, sort_grid = 0;
  if (choose_sort_items(h, n, a.sort_wide != 0, &sort_kernel, &sort_nblk, &sort_grid) != hipSuccess) {
    if (cur != h->device) (void)hipSetDevice(cur);
    return EB_ERR_HIP;
  }
  a.sort_block = kSortThreads * kSortItems[sort_kernel % 4];
  a.sort_nblk_ub = (int32_t)sort_nblk;
  // the keys kernel clears the digit counts and this call's part of the
  // look-back status
  a.zero_words = (int64_t)((L.hist_bytes + 8 * (size_t)L.passes * sort_nblk * ((size_t)1 << L.bits) + 15) / 16);
  // Bags per keys wavefront: the lookup's rule (about sqrt(bags / resident
  // wavefronts)), but at least enough to fit all wavefronts in about one
  // set of resident ones, up to 8.  A keys wavefront spends most of its time
  // waiting for its offsets and first index chunk, so a small batch gains
  // from fewer, longer wavefronts: on MI355X c2's step 0.117 -> 0.114 ms
  // (2 -> 7 bags), c3a's 0.368 -> 0.365 (4 -> 8); past 8 (c4 at 32 rather
  // than 10) it lost 1%.
  int64_t k = 1;
  {
    const int64_t per_slot = num_bags / kResidentWaves;
    while ((k + 1) * (k + 1) <= per_slot) ++k;
    int64_t fill = (num_bags + kResidentWaves - 1) / kResidentWaves;
    fill = fill > 8 ? 8 : fill;
    k = k < fill ? fill : k;
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
  // 2. sort: digit counts, then one pass per digit
  if (e == hipSuccess) {
    const unsigned hgrid = (unsigned)sort_nblk;
    hipLaunchKernelGGL(a.sort_wide ? eb_bwd_sort_hist_kernel<uint64_t> : eb_bwd_sort_hist_kernel<uint32_t>,
                       dim3(hgrid), dim3(kHistThreads), 0, h->stream, a);
    e = hipGetLastError();
  }
  for (int32_t q = 0; q < L.passes && e == hipSuccess; ++q) {
    hipLaunchKernelGGL(kSortPass[sort_kernel], dim3((unsigned)sort_grid), dim3(kSortThreads), 0, h->stream, a, q);
    e = hipGetLastError();
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
    else if (e == hipSuccess && (herr & kErrSortWait)) st = EB_ERR_HIP;
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
