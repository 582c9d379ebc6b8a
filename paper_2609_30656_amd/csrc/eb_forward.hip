// libeb — pooled EmbeddingBag forward for the AMD Instinct MI355X (gfx950).
//
// The operation is the embedding-table lookup stage (sparse_arch) of the
// paper's DLRM study (Sec. IV-A.2): jagged categorical features in, one
// pooled output embedding per (example, feature) out.  The paper finds that
// stage bound by memory bandwidth with almost no arithmetic, so the kernel is
// built around the HBM3E roofline: every byte of a gathered row is fetched
// once with 128-bit loads, converted in registers and summed in fp32; there
// is no matrix-core work because there is no dense contraction.
//
// Execution model:
//   * a wavefront (64 lanes, a workgroup of its own) pools a run of
//     consecutive bags of one table (k bags; each table's last bags in runs
//     of one, dispatched last), walking their index positions as one stream
//     of chunks of up to 64 indices, one coalesced load per chunk, the next
//     chunk's load issued before the current chunk's rows are gathered;
//   * a row is split into 16-byte lane slices; LPR = lanes per row (the next
//     power of two >= row bytes / 16, at most 64), so one wave-wide load
//     fetches RPL = 64 / LPR rows, in straight-line batches of loads;
//   * each lane accumulates its slice in fp32 registers; at a bag's end the
//     RPL row groups are combined by a fixed-order reduce-scatter across lanes
//     and the owning lanes store the pooled vector;
//   * a handle whose tables share one (storage type, LPR) kind launches a body
//     specialised for it; otherwise one launch per storage type switches on
//     each table's LPR;
//   * bags longer than a threshold (1024 lookups unless EB_LONG_BAG says
//     otherwise) are queued by the wavefront that holds them and pooled by a
//     second kernel, cut into segments that run on many workgroups, each
//     segment's indices staged in LDS and split over four wavefronts; the
//     segments' partial sums are added in segment order.  By default this
//     runs for batches of at least 2^23 lookups (below, the second kernel's
//     launch would cost more than 1% of the lookup) or of 64 lookups per bag
//     on average, and for any batch when EB_LONG_BAG is set.
// Rows wider than 1 KiB take several 1 KiB column passes.  This file also
// holds the C ABI's handle creation and the checks shared by the entry points
// that pool.

#include "eb_device.h"

#include <new>

namespace eb {
namespace {

constexpr int kMaxAutoBagsPerWave = 8;  // cap of the lookup's own choice of bags per wavefront

struct FwdArgs {
  const TableMeta *meta;
  GatherCtx ctx;
  const void *indices;
  const void *offsets;
  const float *weights;
  float *out;
  int64_t num_indices;
  int64_t out_ld;
  int32_t num_bags;
  int32_t batch;
  int32_t idx64;
  int32_t mean;
  int32_t bags_per_wave;     // consecutive bags of one table per wavefront (head runs)
  int32_t groups_per_table;  // runs per table: head_groups + tail_groups
  int32_t head_groups;       // runs of bags_per_wave bags at the start of each table
  int32_t tail_groups;       // runs of tail_run bags after them (the table's last bags)
  int32_t tail_run;          // bags per tail run
  int32_t tail_last;         // 1: every table's head runs first, then every tail run
  int32_t head_waves;        // num_tables * head_groups
  int32_t num_waves;         // num_tables * groups_per_table
  int32_t xcd_remap;         // renumber workgroups XCD-contiguously
  int64_t long_len;          // bags with more lookups are queued for the long-bag pass
  int32_t seg_log2;          // that pass pools them in segments of 2^seg_log2 positions
  LongQueue lq;              // the handle's queue (cap 0: no long-bag pass)
};

// Pool bags [g0, g0 + nb) of one table (batch rows b0 ..) over the 1 KiB column
// window starting at byte col_base.  The bags' index positions are walked as
// one stream of chunks of up to 64; the next chunk's indices are loaded before
// the current chunk's rows are gathered, so each chunk costs one memory round
// trip.
// offsets[g0 .. g0 + nb] of a run of bags, one per lane (lanes past nb hold 0)
__device__ __forceinline__ int64_t run_offsets(const FwdArgs &a, int32_t g0, int nb) {
  const int lane = threadIdx.x & (kWave - 1);
  int64_t o = 0;
  if (lane <= nb) {
    o = a.idx64 ? static_cast<const int64_t *>(a.offsets)[g0 + lane]
                : (int64_t) static_cast<const int32_t *>(a.offsets)[g0 + lane];
  }
  return o;
}

// The run of bags wavefront w pools: table t, batch rows [b0, b0 + nb).  A
// table's bags are cut into head runs of bags_per_wave bags followed by tail
// runs of tail_run bags (fewer, so the wavefronts dispatched last hold less
// work and a long power-law bag ends the launch less late).  Wavefront ids
// run table by table, or, with tail_last, through every table's head runs
// before any tail run.
__device__ __forceinline__ void wave_run(const FwdArgs &a, int32_t w, int32_t &t, int32_t &b0, int32_t &nb) {
  int32_t r;
  if (!a.tail_last) {
    t = w / a.groups_per_table;
    r = w - t * a.groups_per_table;
  } else if (w < a.head_waves) {
    t = w / a.head_groups;
    r = w - t * a.head_groups;
  } else {
    const int32_t v = w - a.head_waves;
    t = v / a.tail_groups;
    r = a.head_groups + (v - t * a.tail_groups);
  }
  const bool head = r < a.head_groups;
  const int32_t k = head ? a.bags_per_wave : a.tail_run;
  b0 = head ? r * a.bags_per_wave : a.head_groups * a.bags_per_wave + (r - a.head_groups) * a.tail_run;
  nb = (a.batch - b0) < k ? (a.batch - b0) : k;
}

template <int DT, int LPR, bool W>
__device__ __forceinline__ void pool_bags(const TableMeta &m, const FwdArgs &a, int32_t g0, int nb, int32_t b0,
                                          int col_base, int64_t my_off, uint32_t queued) {
  // my_off: run_offsets(a, g0, nb); bag j is skipped when bit j of `queued`
  // is set (the long-bag pass pools it)
  using R = Reduce<DT, LPR>;
  constexpr int V = Vals<DT>::n;
  const int lane = threadIdx.x & (kWave - 1);
  const int colb = col_base + (lane % LPR) * 16;
  const bool colok = colb < m.code_bytes;
  // bag j's index range, clamped into [0, N) so nothing is read outside the
  // index array whatever the offsets hold (a broken partition is reported)
  auto bag_range = [&](int j, int64_t &lo, int64_t &hi, bool &skip) {
    lo = readlane64(my_off, j);
    hi = readlane64(my_off, j + 1);
    const int32_t g = g0 + j;
    bool bad = lo < 0 || hi < lo || hi > a.num_indices;
    bad |= (g == 0 && lo != 0) || (g == a.num_bags - 1 && hi != a.num_indices);
    if (bad) {
      if (lane == 0) atomicOr(a.ctx.err, kErrOffsets);
      lo = lo < 0 ? 0 : (lo > a.num_indices ? a.num_indices : lo);
      hi = hi < lo ? lo : (hi > a.num_indices ? a.num_indices : hi);
    }
    skip = (queued >> j) & 1u;
    if (skip) hi = lo;
  };

  constexpr bool SPLIT = EB_INT8_SPLIT_BIAS && DT == kU8 && !W;
  float acc[V];
  float cb = 0.0f;
#pragma unroll
  for (int i = 0; i < V; ++i) acc[i] = 0.0f;

  int j = 0;
  int64_t blo, bhi;
  bool bskip;
  bag_range(0, blo, bhi, bskip);
  int64_t c = blo;
  RawChunk cur = load_chunk<W>(a.indices, a.weights, a.idx64, c, bhi);
  while (true) {
    const bool last = c + kWave >= bhi;
    int jn = j;
    int64_t cn = c + kWave, nlo = blo, nhi = bhi;
    bool nskip = bskip;
    if (last) {
      jn = j + 1;
      if (jn < nb) {
        bag_range(jn, nlo, nhi, nskip);
        cn = nlo;
      }
    }
    const bool more = !last || jn < nb;
    RawChunk nxt;
    if (more) nxt = load_chunk<W>(a.indices, a.weights, a.idx64, cn, nhi);

    gather_chunk<DT, LPR, W, SPLIT>(m, a.ctx, resolve(cur, m.num_rows, a.idx64), acc, cb, colb, colok);

    if (last) {
      if constexpr (SPLIT) {
#pragma unroll
        for (int i = 0; i < V; ++i) acc[i] += cb;
        cb = 0.0f;
      }
      R::run(acc);
      if (R::stores(lane) && colok && !bskip) {
        const int64_t L = bhi - blo;
        const int f = R::first_value(lane);
        float outv[R::KEEP];
#pragma unroll
        for (int i = 0; i < R::KEEP; ++i) outv[i] = acc[i];
        if (a.mean && L > 0) {
          const float fl = (float)L;
#pragma unroll
          for (int i = 0; i < R::KEEP; ++i) outv[i] = outv[i] / fl;
        }
        store_slice<R::KEEP>(a.out + (int64_t)(b0 + j) * a.out_ld + m.out_col + colb / Vals<DT>::esize + f, outv);
      }
#pragma unroll
      for (int i = 0; i < V; ++i) acc[i] = 0.0f;
    }
    if (!more) break;
    j = jn;
    c = cn;
    blo = nlo;
    bhi = nhi;
    bskip = nskip;
    cur = nxt;
  }
}

// ----------------------------------------------------------------------------
// Long bags.  One wavefront streaming a bag of many thousand lookups would
// end the launch long after the others, so a wavefront queues its bags of
// more than long_len lookups for a second kernel and skips them:
//   * before its loop, the wavefront finds its long bags from the offsets it
//     holds (the whole run's length from two lane reads, which settles the
//     usual case; for a longer run, one ballot over its bags' lengths), and
//     for each reserves K = ceil(L / seg) consecutive entries of the
//     handle's queue with one atomic add, writing the bag's id and first
//     entry into them.  A bag whose entries do not fit the queue is pooled
//     by the wavefront as usual;
//   * the long-bag pass (eb_long_pass_kernel) runs after the lookup on the
//     same stream.  Its workgroups of four wavefronts take one entry (a
//     segment of seg positions) at a time from an atomic head: stage the
//     segment's indices (and weights) in LDS with coalesced loads, let each
//     wavefront pool a quarter of them with the lookup's row gather, and add
//     the four partial vectors in LDS in wavefront order into the entry's
//     partial row.  The workgroup whose arrival completes the bag adds its K
//     partial rows in segment order (so the result does not depend on
//     scheduling), divides by L for mean pooling and stores the bag.  The
//     last workgroup out clears the queue's counters for the next call.
// No workgroup waits for another.  Every value that decides the pass's
// control flow around its barriers is made wave-uniform (readfirstlane): a
// loop whose exit the compiler takes for divergent may be laid out so that
// thread 0's work at the end of one round and at the start of the next sit
// outside the loop the other threads re-enter, and they then read the shared
// entry word before thread 0 has written it.

constexpr int kLongBlocks = 256;          // workgroups of the long-bag pass (one per CU)
constexpr uint32_t kNoBag = 0xFFFFFFFFu;   // an entry of a reservation that did not fit

__device__ __forceinline__ uint32_t agent_load(const uint32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void agent_store(uint32_t *p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t agent_add(uint32_t *p, uint32_t v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int64_t uniform64(int64_t v) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Queue the run's bags of more than a.long_len lookups (bags [g0, g0 + nb),
// offsets my_off as run_offsets gives them).  Returns the mask of the bags
// queued; their lengths are taken as pool_bags clamps them.
__device__ __forceinline__ uint32_t queue_long_bags(const FwdArgs &a, int32_t g0, int nb, int64_t my_off) {
  // no bag of the run can be long if the whole run is not (the usual case:
  // two lane reads and a compare); broken offsets go on to the full test
  const int64_t run_lo = readlane64(my_off, 0), run_hi = readlane64(my_off, nb);
  if (run_lo >= 0 && run_hi >= run_lo && run_hi - run_lo <= a.long_len) return 0u;
  const int lane = threadIdx.x & (kWave - 1);
  const int src = lane + 1 < kWave ? lane + 1 : lane;
  const uint32_t nlo = (uint32_t)__shfl((int)(uint32_t)my_off, src);
  const uint32_t nhi = (uint32_t)__shfl((int)(uint32_t)((uint64_t)my_off >> 32), src);
  const int64_t next = (int64_t)(((uint64_t)nhi << 32) | nlo);
  const int64_t lo = my_off < 0 ? 0 : (my_off > a.num_indices ? a.num_indices : my_off);
  const int64_t hi = next < lo ? lo : (next > a.num_indices ? a.num_indices : next);
  const int64_t len = hi - lo;
  uint64_t longm = __ballot(lane < nb && len > a.long_len);
  uint32_t queued = 0;
  while (longm) {
    const int j = __builtin_ctzll(longm);
    longm &= longm - 1;
    const int64_t L = readlane64(len, j);
    const uint32_t K = (uint32_t)((L + ((int64_t)1 << a.seg_log2) - 1) >> a.seg_log2);
    uint32_t s0 = 0;
    if (lane == 0) s0 = agent_add(a.lq.ctrl + kLqTail, K);
    s0 = __builtin_amdgcn_readfirstlane(s0);
    const uint64_t cap = (uint64_t)a.lq.cap;
    const bool fits = (uint64_t)s0 + K <= cap;
    for (uint32_t k = lane; k < K && (uint64_t)s0 + k < cap; k += kWave) {
      a.lq.bag[s0 + k] = fits ? (uint32_t)(g0 + j) : kNoBag;
      a.lq.first[s0 + k] = s0;
    }
    if (fits) queued |= 1u << j;
  }
  return queued;
}

template <int DT, int LPR, bool W>
__device__ __forceinline__ void pool_all_passes(const TableMeta &m, const FwdArgs &a, int32_t g0, int nb,
                                                int32_t b0, int64_t my_off, uint32_t queued) {
  if constexpr (LPR == kWave) {
    for (int p = 0; p < m.passes; ++p) pool_bags<DT, LPR, W>(m, a, g0, nb, b0, p * kPassBytes, my_off, queued);
  } else {
    pool_bags<DT, LPR, W>(m, a, g0, nb, b0, 0, my_off, queued);
  }
}

#define EB_LPR(LOG2)                                                          \
  case LOG2:                                                                  \
    pool_all_passes<DT, (1 << (LOG2)), W>(m, a, g0, nb, b0, my_off, queued);  \
    break;

// One wavefront per run of bags.  DT is the storage type the launch serves
// (wavefronts of other tables skip their own bags).  LOG2 >= 0 fixes the
// lanes per row for handles whose tables all share one kind; LOG2 < 0
// switches on each table's lanes per row.  Specialising keeps the register
// count (and so the occupancy) at what that kind needs.  The fp16 and
// unweighted fp32 kernels that switch over every width are held to 8 waves
// per SIMD (64 VGPRs), which they meet without spilling; the int8 one would
// spill, so it keeps the compiler's choice.  The unweighted int8 kernels of
// one width are held to 8 as well: left alone the compiler gives them 69-72
// VGPRs (7 waves), held they take 50-60 without spilling, and 64 int8 tables
// of 128 values at batch 65 536 run 0.7% faster.
template <int DT, int LOG2, bool W>
__global__ __launch_bounds__(kWave)
__attribute__((amdgpu_waves_per_eu(((LOG2 < 0 && (DT == kF16 || (DT == kF32 && !W))) || (DT == kU8 && LOG2 >= 0 && !W))
                                       ? 8
                                       : 1,
                                   8)))
void eb_pool_kernel(FwdArgs a) {
  const uint32_t blk = a.xcd_remap ? xcd_contiguous(blockIdx.x, gridDim.x) : blockIdx.x;
  const int32_t wid = (int32_t)blk;
  if (wid < a.num_waves) {
    int32_t t, b0, nb;
    wave_run(a, wid, t, b0, nb);
    const int32_t g0 = t * a.batch + b0;
    // the offsets' address needs no table descriptor: issue that load first
    const int64_t my_off = run_offsets(a, g0, nb);
    const TableMeta m = a.meta[t];
    if (m.kind / 8 == DT) {
      const uint32_t queued = a.lq.cap > 0 ? queue_long_bags(a, g0, nb, my_off) : 0u;
      if constexpr (LOG2 >= 0) {
        pool_all_passes<DT, (1 << (LOG2 >= 0 ? LOG2 : 0)), W>(m, a, g0, nb, b0, my_off, queued);
      } else {
        switch (m.kind % 8) {
          EB_LPR(0) EB_LPR(1) EB_LPR(2) EB_LPR(3) EB_LPR(4) EB_LPR(5) EB_LPR(6)
          default:
            break;
        }
      }
    }
  }
}

#undef EB_LPR

// offsets[g], clamped into [0, N] (wave-uniform)
__device__ __forceinline__ int64_t clamped_offset(const FwdArgs &a, int64_t g) {
  const int64_t v = uniform64(a.idx64 ? static_cast<const int64_t *>(a.offsets)[g]
                                      : (int64_t) static_cast<const int32_t *>(a.offsets)[g]);
  return v < 0 ? 0 : (v > a.num_indices ? a.num_indices : v);
}

// Bag g's index range, clamped as pool_bags clamps it (wave-uniform).
__device__ __forceinline__ void long_bag_range(const FwdArgs &a, int64_t g, int64_t &lo, int64_t &hi) {
  lo = clamped_offset(a, g);
  hi = clamped_offset(a, g + 1);
  hi = hi < lo ? lo : hi;
}

// Stage positions [plo, plo + n) of the index stream (and their weights) in
// LDS, indices widened to 64 bits.
template <bool W>
__device__ __forceinline__ void stage_segment(const FwdArgs &a, int64_t plo, int n, int64_t *s_idx, float *s_w) {
  for (int i = threadIdx.x; i < n; i += kBlock) {
    s_idx[i] = a.idx64 ? static_cast<const int64_t *>(a.indices)[plo + i]
                       : (int64_t) static_cast<const int32_t *>(a.indices)[plo + i];
    if constexpr (W) s_w[i] = a.weights[plo + i];
  }
  __syncthreads();
}

// The workgroup pools the n staged positions of one segment of a table-m bag:
// wavefront w takes the w-th contiguous quarter of the segment's 64-position
// chunks.  Per 1 KiB column window, the wavefronts' reduced vectors meet in
// s_part and their sum, in wavefront order, is written to dst (the row's
// first m.dim values).
template <int DT, int LPR, bool W>
__device__ __forceinline__ void long_segment(const TableMeta &m, const FwdArgs &a, const int64_t *s_idx,
                                             const float *s_w, int n, float *s_part, float *dst) {
  using R = Reduce<DT, LPR>;
  constexpr int V = Vals<DT>::n;
  constexpr int WIN = kPassBytes / Vals<DT>::esize;  // values per column window
  constexpr bool SPLIT = EB_INT8_SPLIT_BIAS && DT == kU8 && !W;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int chunks = (n + kWave - 1) / kWave;
  const int per = (chunks + kWavesPerBlock - 1) / kWavesPerBlock;
  const int c0 = wave * per < chunks ? wave * per : chunks;
  const int c1 = c0 + per < chunks ? c0 + per : chunks;
  const int passes = LPR == kWave ? m.passes : 1;
  for (int p = 0; p < passes; ++p) {
    const int colb = p * kPassBytes + (lane % LPR) * 16;
    const bool colok = colb < m.code_bytes;
    float acc[V];
    float cb = 0.0f;
#pragma unroll
    for (int i = 0; i < V; ++i) acc[i] = 0.0f;
    for (int c = c0; c < c1; ++c) {
      RawChunk k;
      k.n = n - c * kWave < kWave ? n - c * kWave : kWave;
      const int at = c * kWave + (lane < k.n ? lane : 0);
      const uint64_t v = (uint64_t)s_idx[at];
      k.lo = (uint32_t)v;
      k.hi = (uint32_t)(v >> 32);
      k.w = W ? s_w[at] : 0.0f;
      gather_chunk<DT, LPR, W, SPLIT>(m, a.ctx, resolve(k, m.num_rows, 1), acc, cb, colb, colok);
    }
    if constexpr (SPLIT) {
#pragma unroll
      for (int i = 0; i < V; ++i) acc[i] += cb;
    }
    R::run(acc);
    if (R::stores(lane)) {
      const int e = (lane % LPR) * V + R::first_value(lane);
#pragma unroll
      for (int i = 0; i < R::KEEP; ++i) s_part[wave * WIN + e + i] = acc[i];
    }
    __syncthreads();
    const int rest = (m.code_bytes - p * kPassBytes) / Vals<DT>::esize;
    const int cols = rest < WIN ? rest : WIN;
    for (int c = threadIdx.x; c < cols; c += kBlock) {
      float v = s_part[c];
#pragma unroll
      for (int w = 1; w < kWavesPerBlock; ++w) v += s_part[w * WIN + c];
      dst[p * WIN + c] = v;
    }
    __syncthreads();  // s_part is reused by the next window
  }
}

// The long-bag pass for the lookup's storage type DT (see above).
template <int DT, bool W>
__global__ __launch_bounds__(kBlock) void eb_long_pass_kernel(FwdArgs a) {
  constexpr int WIN = kPassBytes / Vals<DT>::esize;
  __shared__ int64_t s_idx[kLongSegMax];
  __shared__ float s_w[W ? kLongSegMax : 1];
  __shared__ float s_part[kWavesPerBlock * WIN];
  __shared__ uint32_t s_word;
  uint32_t *ctrl = a.lq.ctrl;
  const uint32_t tail = __builtin_amdgcn_readfirstlane(agent_load(ctrl + kLqTail));
  if (tail == 0) return;  // nothing queued (the usual case): nothing to clear either
  const int tid = threadIdx.x;
  const int64_t seg = (int64_t)1 << a.seg_log2;
  const uint32_t cap = (uint32_t)a.lq.cap;
  const uint32_t end = tail < cap ? tail : cap;
  // one entry per round; `end` entries in all, so no workgroup takes more
  for (uint32_t round = 0; round <= end; ++round) {
    if (tid == 0) s_word = agent_add(ctrl + kLqHead, 1);
    __syncthreads();
    const uint32_t e = __builtin_amdgcn_readfirstlane(s_word);
    __syncthreads();  // s_word is rewritten only after every thread has read it
    if (e >= end) break;
    const uint32_t gu = __builtin_amdgcn_readfirstlane(a.lq.bag[e]);
    if (gu == kNoBag) continue;  // part of a reservation that did not fit
    const uint32_t s0 = __builtin_amdgcn_readfirstlane(a.lq.first[e]);
    int64_t lo, hi;
    long_bag_range(a, gu, lo, hi);
    const int64_t L = hi - lo;
    const uint32_t K = (uint32_t)((L + seg - 1) >> a.seg_log2);
    const int64_t plo = lo + (int64_t)(e - s0) * seg;
    const int n = (int)((plo + seg < hi ? plo + seg : hi) - plo);
    const int32_t t = (int32_t)(gu / (uint32_t)a.batch);
    const int32_t b = (int32_t)(gu - (uint32_t)t * (uint32_t)a.batch);
    const TableMeta m = a.meta[t];
    stage_segment<W>(a, plo, n, s_idx, s_w);
    float *part = a.lq.part + (size_t)e * a.lq.part_ld;
    switch (m.kind % 8) {
      case 0: long_segment<DT, 1, W>(m, a, s_idx, s_w, n, s_part, part); break;
      case 1: long_segment<DT, 2, W>(m, a, s_idx, s_w, n, s_part, part); break;
      case 2: long_segment<DT, 4, W>(m, a, s_idx, s_w, n, s_part, part); break;
      case 3: long_segment<DT, 8, W>(m, a, s_idx, s_w, n, s_part, part); break;
      case 4: long_segment<DT, 16, W>(m, a, s_idx, s_w, n, s_part, part); break;
      case 5: long_segment<DT, 32, W>(m, a, s_idx, s_w, n, s_part, part); break;
      case 6: long_segment<DT, 64, W>(m, a, s_idx, s_w, n, s_part, part); break;
      default: break;
    }
    __threadfence();  // this segment's partial row is visible before it is counted
    if (tid == 0) s_word = agent_add(a.lq.arrived + s0, 1);
    __syncthreads();
    const bool last = __builtin_amdgcn_readfirstlane(s_word) == K - 1;
    __syncthreads();
    if (last) {
      __threadfence();  // the bag's other partial rows are visible here
      const float *p0 = a.lq.part + (size_t)s0 * a.lq.part_ld;
      float *dst = a.out + (int64_t)b * a.out_ld + m.out_col;
      for (int c = tid; c < m.dim; c += kBlock) {
        // the partial rows in segment order, eight loads in flight
        float v = 0.0f;
        for (uint32_t k = 0; k < K; k += 8) {
          float x[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) x[u] = k + u < K ? p0[(size_t)(k + u) * a.lq.part_ld + c] : 0.0f;
#pragma unroll
          for (int u = 0; u < 8; ++u)
            if (k + u < K) v += x[u];
        }
        if (a.mean && L > 0) v = v / (float)L;
        __builtin_nontemporal_store(v, dst + c);
      }
      if (tid == 0) agent_store(a.lq.arrived + s0, 0u);  // cleared for the next call
    }
  }
  // the last workgroup out clears the counters (every workgroup has left the
  // loop by then, so none reads them again)
  if (tid == 0 && agent_add(ctrl + kLqFinished, 1) == gridDim.x - 1) {
    agent_store(ctrl + kLqTail, 0u);
    agent_store(ctrl + kLqHead, 0u);
    agent_store(ctrl + kLqFinished, 0u);
  }
}

typedef void (*KernelFn)(FwdArgs);

// kernel for (storage type, log2 lanes per row or -1, weighted)
template <int DT, bool W>
KernelFn pick_kernel(int log2) {
  switch (log2) {
    case 0: return eb_pool_kernel<DT, 0, W>;
    case 1: return eb_pool_kernel<DT, 1, W>;
    case 2: return eb_pool_kernel<DT, 2, W>;
    case 3: return eb_pool_kernel<DT, 3, W>;
    case 4: return eb_pool_kernel<DT, 4, W>;
    case 5: return eb_pool_kernel<DT, 5, W>;
    case 6: return eb_pool_kernel<DT, 6, W>;
    default: return eb_pool_kernel<DT, -1, W>;
  }
}

KernelFn pick_kernel(int dt, int log2, bool weighted) {
  if (dt == kF32) return weighted ? pick_kernel<kF32, true>(log2) : pick_kernel<kF32, false>(log2);
  if (dt == kF16) return weighted ? pick_kernel<kF16, true>(log2) : pick_kernel<kF16, false>(log2);
  return weighted ? pick_kernel<kU8, true>(log2) : pick_kernel<kU8, false>(log2);
}

KernelFn pick_long_kernel(int dt, bool weighted) {
  if (dt == kF32) return weighted ? eb_long_pass_kernel<kF32, true> : eb_long_pass_kernel<kF32, false>;
  if (dt == kF16) return weighted ? eb_long_pass_kernel<kF16, true> : eb_long_pass_kernel<kF16, false>;
  return weighted ? eb_long_pass_kernel<kU8, true> : eb_long_pass_kernel<kU8, false>;
}

}  // namespace
}  // namespace eb

namespace eb {

eb_status check_forward_args(const eb_tables *h, const eb_tensor &indices, const eb_tensor &offsets,
                             const eb_tensor &weights, eb_pooling pooling, const eb_tensor &out, FwdShape *sh) {
  if (!h) return EB_ERR_INVALID_ARG;
  if (indices.elem_type != EB_I32 && indices.elem_type != EB_I64) return EB_ERR_DTYPE;
  if (offsets.elem_type != indices.elem_type) return EB_ERR_DTYPE;
  if (out.elem_type != EB_T_F32) return EB_ERR_DTYPE;
  if (pooling != EB_POOL_SUM && pooling != EB_POOL_MEAN) return EB_ERR_INVALID_ARG;
  if (!offsets.data || !out.data) return EB_ERR_INVALID_ARG;
  if (indices.numel < 0 || (indices.numel > 0 && !indices.data)) return EB_ERR_INVALID_ARG;
  const bool weighted = weights.data != nullptr;
  if (weighted) {
    if (weights.elem_type != EB_T_F32) return EB_ERR_DTYPE;
    if (pooling == EB_POOL_MEAN) return EB_ERR_INVALID_ARG;
    if (weights.numel != indices.numel) return EB_ERR_SHAPE;
  }
  if (offsets.numel < 2 || (offsets.numel - 1) % h->num_tables != 0) return EB_ERR_SHAPE;
  const int64_t num_bags = offsets.numel - 1;
  const int64_t batch = num_bags / h->num_tables;
  if (num_bags > INT32_MAX) return EB_ERR_SHAPE;
  if (out.numel != batch * h->sum_dim) return EB_ERR_SHAPE;
  const size_t isz = indices.elem_type == EB_I64 ? 8 : 4;
  if (reinterpret_cast<uintptr_t>(out.data) % 16 != 0 || reinterpret_cast<uintptr_t>(offsets.data) % isz != 0 ||
      reinterpret_cast<uintptr_t>(indices.data) % isz != 0 ||
      (weighted && reinterpret_cast<uintptr_t>(weights.data) % 4 != 0))
    return EB_ERR_UNSUPPORTED;
  sh->num_bags = num_bags;
  sh->batch = batch;
  sh->weighted = weighted;
  return EB_OK;
}

hipError_t launch_forward(const eb_tables *h, const eb_tensor &indices, const eb_tensor &offsets,
                          const eb_tensor &weights, eb_pooling pooling, const eb_tensor &out, const FwdShape &sh) {
  FwdArgs a;
  a.meta = h->d_meta;
  a.indices = indices.data;
  a.offsets = offsets.data;
  a.weights = static_cast<const float *>(weights.data);
  a.out = static_cast<float *>(const_cast<void *>(out.data));
  a.ctx.err = h->d_err;
  a.ctx.zero = h->d_zero;
  a.ctx.one = 1.0f;
  a.xcd_remap = h->xcd_remap;
  a.long_len = h->long_bag_len > 0 ? h->long_bag_len : INT64_MAX;  // 0: no long-bag pass
  a.seg_log2 = h->long_seg_log2;
  a.lq = h->lq;
  // The pass costs one more kernel on the stream whether or not a bag needs
  // it (on MI355X 1.7-6 us: 8% of a 23 us lookup of a million lookups in
  // bags of twenty, under 1% from about eight million lookups), so unless
  // the handle asked for it (EB_LONG_BAG set) it runs for batches that large,
  // and for batches whose bags hold kLongPassMinMean lookups or more on
  // average: bag lengths are long-tailed, so those are the batches that hold
  // bags of thousands.
  const bool long_pass = h->lq.cap > 0 && (h->long_bag_forced || indices.numel >= kLongPassMinLookups ||
                                           indices.numel >= kLongPassMinMean * sh.num_bags);
  if (!long_pass) a.lq.cap = 0;  // the lookup queues nothing: every bag is its wavefront's
  a.num_indices = indices.numel;
  a.out_ld = h->sum_dim;
  a.num_bags = (int32_t)sh.num_bags;
  a.batch = (int32_t)sh.batch;
  a.idx64 = indices.elem_type == EB_I64;
  a.mean = pooling == EB_POOL_MEAN;
  int64_t k = h->bags_per_wave;
  if (k == 0) {
    // More bags per wavefront hide more latency (each bag's indices arrive
    // while the previous bag's rows are in flight); fewer leave more
    // wavefronts to balance the load.  Measured optimum on MI355X: about
    // sqrt(bags / resident wavefronts), at most 8 (with the taper below, 8
    // beat that rule's 10 on 100 mixed fp16 tables at batch 8192 by 1.5%,
    // and its 22 on 64 int8 tables at batch 65536 by 3%).
    const int64_t per_slot = sh.num_bags / kResidentWaves;
    k = 1;
    while ((k + 1) * (k + 1) <= per_slot) ++k;
    k = k > kMaxAutoBagsPerWave ? kMaxAutoBagsPerWave : k;
  }
  a.bags_per_wave = (int32_t)k;
  // Taper: the last bags of each table go in runs of tail_run bags, enough of
  // them for kTailGens full sets of resident wavefronts over all tables; the
  // rest in runs of k.  Long runs first and short ones last end the launch
  // sooner when bag lengths are heavy-tailed (on MI355X, 8 fp16 tables at
  // batch 16384 with power-law lengths on 1..200: 6-10% faster at 4 sets).  With k <= 2 the runs are short
  // already and a taper only adds wavefronts.  A handle made with
  // EB_TAIL_BAGS set uses that many tail bags per table instead.
  const int64_t run = h->tail_run < k ? h->tail_run : k;
  int64_t tail_bags = h->tail_bags >= 0 ? h->tail_bags
                      : (k >= 3 ? (kTailGens * kResidentWaves * run + h->num_tables - 1) / h->num_tables : 0);
  tail_bags = tail_bags < sh.batch ? tail_bags : sh.batch;
  const int64_t tail_run = tail_bags > 0 ? run : k;
  const int64_t head_groups = (sh.batch - tail_bags) / k;
  const int64_t rest = sh.batch - head_groups * k;
  a.head_groups = (int32_t)head_groups;
  a.tail_run = (int32_t)tail_run;
  a.tail_groups = (int32_t)((rest + tail_run - 1) / tail_run);
  a.groups_per_table = a.head_groups + a.tail_groups;
  // Without the XCD renumbering the launch runs its wavefronts in id order,
  // so the tail runs of every table go last; with it, each XCD runs its own
  // contiguous range of tables and a table's tail runs end that table.
  a.tail_last = (tail_bags > 0 && !h->xcd_remap && head_groups > 0 && a.tail_groups > 0) ? 1 : 0;
  a.head_waves = (int32_t)(head_groups * h->num_tables);
  const int64_t num_waves = (int64_t)a.groups_per_table * h->num_tables;
  a.num_waves = (int32_t)num_waves;

  hipError_t e = hipSuccess;
  std::lock_guard<std::mutex> lock(*h->enqueue);
  // one launch per storage type present (one in the usual case), each
  // followed by the long-bag pass over what it queued
  for (int dt = 0; dt < 3 && e == hipSuccess; ++dt) {
    if (!(h->dtype_mask & (1 << dt))) continue;
    hipLaunchKernelGGL(pick_kernel(dt, h->single_log2, sh.weighted), dim3((unsigned)num_waves), dim3(kWave), 0,
                       h->stream, a);
    e = hipGetLastError();
    if (e == hipSuccess && long_pass) {
      hipLaunchKernelGGL(pick_long_kernel(dt, sh.weighted), dim3(kLongBlocks), dim3(kBlock), 0, h->stream, a);
      e = hipGetLastError();
    }
  }
  return e;
}

// Whether kernels on device `dev` can read memory at p: that device's own
// memory, managed memory or pinned host memory (not pageable host memory, and
// not another device's memory).
static bool device_can_read(const void *p, int dev) {
  hipPointerAttribute_t at;
  if (hipPointerGetAttributes(&at, p) != hipSuccess) {
    (void)hipGetLastError();  // an unknown pointer leaves the error behind
    return false;
  }
  if (at.type == hipMemoryTypeDevice) return at.device == dev;
  return at.type == hipMemoryTypeManaged || at.type == hipMemoryTypeHost || at.type == hipMemoryTypeUnified;
}

hipError_t begin_checked(const eb_tables *h) {
  return h->checked ? hipMemsetAsync(h->d_err, 0, sizeof(int), h->stream) : hipSuccess;
}

eb_status end_checked(const eb_tables *h, hipError_t e) {
  eb_status st = EB_OK;
  if (e == hipSuccess && h->checked) {
    int herr = 0;
    e = hipMemcpyAsync(&herr, h->d_err, sizeof(int), hipMemcpyDeviceToHost, h->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h->stream);
    if (e == hipSuccess && (herr & kErrOffsets)) st = EB_ERR_OFFSETS;
    else if (e == hipSuccess && (herr & kErrIndex)) st = EB_ERR_INDEX_OOB;
    else if (e == hipSuccess && (herr & kErrOutSize)) st = EB_ERR_SHAPE;
  }
  return e != hipSuccess ? EB_ERR_HIP : st;
}

}  // namespace eb

using namespace eb;

extern "C" {

const char *eb_status_string(eb_status s) {
  switch (s) {
    case EB_OK: return "ok";
    case EB_ERR_INVALID_ARG: return "invalid argument";
    case EB_ERR_DTYPE: return "unknown or mismatched data type";
    case EB_ERR_SHAPE: return "sizes do not fit together";
    case EB_ERR_UNSUPPORTED: return "unsupported dimension or alignment";
    case EB_ERR_INDEX_OOB: return "index outside its table (checked mode)";
    case EB_ERR_OFFSETS: return "offsets are not a partition of the indices (checked mode)";
    case EB_ERR_OOM: return "device allocation failed";
    case EB_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

eb_status eb_create_tables(const eb_table_desc *descs, int32_t num_tables, void *hip_stream, eb_tables **out) {
  if (!out) return EB_ERR_INVALID_ARG;
  *out = nullptr;
  if (!descs || num_tables < 1 || num_tables > 65535) return EB_ERR_INVALID_ARG;

  TableMeta *meta = static_cast<TableMeta *>(calloc((size_t)num_tables, sizeof(TableMeta)));
  if (!meta) return EB_ERR_OOM;
  int64_t col = 0, rows_before = 0;
  uint64_t key_before = 0;
  eb_status st = EB_OK;
  for (int32_t t = 0; t < num_tables && st == EB_OK; ++t) {
    const eb_table_desc &d = descs[t];
    int esize, align, dim_mult;
    if (d.dtype == EB_F32) {
      esize = 4; align = 16; dim_mult = 4;
    } else if (d.dtype == EB_F16) {
      esize = 2; align = 16; dim_mult = 8;
    } else if (d.dtype == EB_INT8_ROWWISE) {
      esize = 1; align = 4; dim_mult = 16;
    } else if (d.dtype == EB_INT8_ROWWISE_SPLIT) {
      esize = 1; align = 16; dim_mult = 16;
    } else {
      st = EB_ERR_DTYPE;
      break;
    }
    const int64_t code_bytes = (int64_t)d.dim * esize;
    const int64_t row_bytes = code_bytes + (d.dtype == EB_INT8_ROWWISE ? 4 : 0);
    if (!d.data || d.num_rows < 1 || d.num_rows > INT32_MAX || d.dim < 1 || d.dim > kMaxDim ||
        d.row_stride_bytes < row_bytes) {
      st = EB_ERR_INVALID_ARG;
    } else if (d.dim % dim_mult != 0 || d.row_stride_bytes % align != 0 ||
               reinterpret_cast<uintptr_t>(d.data) % align != 0 || d.row_stride_bytes > INT32_MAX) {
      st = EB_ERR_UNSUPPORTED;
    } else {
      TableMeta &m = meta[t];
      m.data = static_cast<const unsigned char *>(d.data);
      m.row_stride = (uint32_t)d.row_stride_bytes;
      m.num_rows = (int32_t)d.num_rows;
      m.dim = d.dim;
      m.code_bytes = (int32_t)code_bytes;
      m.out_col = (int32_t)col;
      // both int8 row-wise layouts run the int8 kernels; they differ only in
      // where a row's scale/bias word is
      const int kernel_dt = d.dtype == EB_INT8_ROWWISE_SPLIT ? kU8 : d.dtype;
      m.kind = kernel_dt * 8 + log2_lanes_per_row((int)code_bytes);
      if (d.dtype == EB_INT8_ROWWISE_SPLIT) {
        m.sb_base = m.data + (size_t)d.num_rows * (size_t)d.row_stride_bytes;
        m.sb_stride = 4;
      } else {
        m.sb_base = m.data + code_bytes;
        m.sb_stride = m.row_stride;
      }
      m.passes = (int32_t)((code_bytes + kPassBytes - 1) / kPassBytes);
      m.state_base = rows_before;
      m.key_base = (uint32_t)(key_before <= UINT32_MAX ? key_before : 0);
      rows_before += d.num_rows;
      key_before += d.num_rows + 1;
      col += d.dim;
      if (col > INT32_MAX) st = EB_ERR_SHAPE;
    }
  }
  if (st != EB_OK) {
    free(meta);
    return st;
  }

  eb_tables *h = static_cast<eb_tables *>(calloc(1, sizeof(eb_tables)));
  if (!h) {
    free(meta);
    return EB_ERR_OOM;
  }
  if (hipGetDevice(&h->device) != hipSuccess) {
    free(meta);
    free(h);
    return EB_ERR_HIP;
  }
  // the kernels read the rows in place: refuse memory this device cannot reach
  for (int32_t t = 0; t < num_tables; ++t) {
    if (!device_can_read(descs[t].data, h->device)) {
      free(meta);
      free(h);
      return EB_ERR_INVALID_ARG;
    }
  }
  h->stream = static_cast<hipStream_t>(hip_stream);
  h->num_tables = num_tables;
  h->dtype_mask = 0;
  h->single_log2 = meta[0].kind % 8;
  h->max_dim = 0;
  h->uniform_dim = meta[0].dim;
  h->total_rows = rows_before;
  // the backward sorts (table, row) as one 32-bit key: sum of (rows + 1) must fit
  h->backward_ok = key_before <= (uint64_t)UINT32_MAX;
  for (int32_t t = 0; t < num_tables; ++t) {
    h->dtype_mask |= 1 << (meta[t].kind / 8);
    if (meta[t].kind != meta[0].kind) h->single_log2 = -1;
    if (meta[t].dim > h->max_dim) h->max_dim = meta[t].dim;
    if (meta[t].dim != meta[0].dim) h->uniform_dim = 0;
    if (meta[t].kind / 8 == kU8 || meta[t].dim > kMaxBackwardDim) h->backward_ok = 0;
  }
  h->sum_dim = col;
  const char *chk = getenv("EB_CHECK");
  h->checked = (chk && chk[0] == '1') ? 1 : 0;
  const char *remap = getenv("EB_XCD_REMAP");
  h->xcd_remap = remap ? (remap[0] == '1') : (num_tables <= kRemapMaxTables);
  const char *bremap = getenv("EB_BWD_XCD_REMAP");
  h->bwd_xcd_remap = bremap ? (bremap[0] == '1') : (num_tables <= kRemapMaxTables);
  const char *btc = getenv("EB_BWD_TILE_CHUNKS");
  h->bwd_tile_chunks = btc ? atoi(btc) : 0;
  if (h->bwd_tile_chunks < 0 || h->bwd_tile_chunks > 16) h->bwd_tile_chunks = 0;
  const char *bsi = getenv("EB_BWD_SORT_ITEMS");
  h->bwd_sort_items = bsi ? atoi(bsi) : 0;
  if (h->bwd_sort_items != 4 && h->bwd_sort_items != 8 && h->bwd_sort_items != 12 && h->bwd_sort_items != 16)
    h->bwd_sort_items = 0;
  const char *lb = getenv("EB_LONG_BAG");
  h->long_bag_len = lb ? atoll(lb) : kDefaultLongBag;
  if (h->long_bag_len < 0) h->long_bag_len = kDefaultLongBag;
  h->long_bag_forced = lb && h->long_bag_len > 0;
  // positions per long-bag segment: a power of two from 64 to kLongSegMax
  const char *ls = getenv("EB_LONG_SEG");
  int64_t seg = ls ? atoll(ls) : kDefaultLongSeg;
  if (seg < kWave || seg > kLongSegMax) seg = kDefaultLongSeg;
  h->long_seg_log2 = 0;
  while ((2LL << h->long_seg_log2) <= seg) ++h->long_seg_log2;
  const char *tb = getenv("EB_TAIL_BAGS");
  h->tail_bags = tb ? atoll(tb) : -1;
  if (h->tail_bags < -1) h->tail_bags = -1;
  const char *tr = getenv("EB_TAIL_RUN");
  h->tail_run = tr ? atoi(tr) : 1;
  if (h->tail_run < 1 || h->tail_run > kMaxBagsPerWave) h->tail_run = 1;
  const char *bpw = getenv("EB_BAGS_PER_WAVE");
  h->bags_per_wave = bpw ? atoi(bpw) : 0;
  if (h->bags_per_wave < 0 || h->bags_per_wave > kMaxBagsPerWave) h->bags_per_wave = 0;

  const size_t meta_bytes = sizeof(TableMeta) * (size_t)num_tables;
  // [descriptors][error word, padded to 256 B][zero row][long-bag queue]
  const size_t err_off = (meta_bytes + 255) / 256 * 256;
  const size_t zero_off = err_off + 256;
  const size_t lq_off = (zero_off + kZeroBytes + 255) / 256 * 256;
  // the long-bag queue: 256 B of counters, then per entry a bag id, a first
  // entry and an arrival count, then one partial row of the widest table per
  // entry (kLqMaxPartialFloats floats at most)
  const int32_t part_ld = (h->max_dim + 3) / 4 * 4;
  int64_t lq_cap = h->long_bag_len > 0 ? kLqMaxPartialFloats / part_ld : 0;
  lq_cap = lq_cap > kLqMaxEntries ? kLqMaxEntries : lq_cap;
  const size_t lq_part_off = (256 + (size_t)lq_cap * 12 + 255) / 256 * 256;
  const size_t lq_bytes = lq_cap > 0 ? lq_part_off + (size_t)lq_cap * part_ld * 4 : 0;
  const size_t total = lq_off + lq_bytes;
  // a caller's cap on the handle's device memory: past it, fail as the
  // allocator would
  const char *cap = getenv("EB_DEVICE_ALLOC_LIMIT");
  if (cap && cap[0] && strtoull(cap, nullptr, 10) < total) {
    free(meta);
    free(h);
    return EB_ERR_OOM;
  }
  h->enqueue = new (std::nothrow) std::mutex();
  if (!h->enqueue) {
    free(meta);
    free(h);
    return EB_ERR_OOM;
  }
  void *dev = nullptr;
  hipError_t e = hipMalloc(&dev, total);
  if (e != hipSuccess) {
    delete h->enqueue;
    free(meta);
    free(h);
    return e == hipErrorOutOfMemory ? EB_ERR_OOM : EB_ERR_HIP;
  }
  h->d_meta = static_cast<TableMeta *>(dev);
  h->d_err = reinterpret_cast<int *>(static_cast<char *>(dev) + err_off);
  h->d_zero = static_cast<unsigned char *>(dev) + zero_off;
  h->lq = LongQueue{};
  if (lq_cap > 0) {
    char *q = static_cast<char *>(dev) + lq_off;
    h->lq.ctrl = reinterpret_cast<uint32_t *>(q);
    h->lq.bag = reinterpret_cast<uint32_t *>(q + 256);
    h->lq.first = h->lq.bag + lq_cap;
    h->lq.arrived = h->lq.first + lq_cap;
    h->lq.part = reinterpret_cast<float *>(q + lq_part_off);
    h->lq.cap = (int32_t)lq_cap;
    h->lq.part_ld = part_ld;
  } else {
    h->long_bag_len = 0;  // no queue: no bag is left to the long-bag pass
  }
  e = hipMemcpy(h->d_meta, meta, meta_bytes, hipMemcpyHostToDevice);
  // the error word, the zero row, the queue's counters and arrival counts
  // start at zero (its entries and partial rows are written before they are
  // read); the copies and clears end before this call returns
  if (e == hipSuccess) e = hipMemset(static_cast<char *>(dev) + err_off, 0, 256 + kZeroBytes);
  if (e == hipSuccess && lq_cap > 0) e = hipMemset(h->lq.ctrl, 0, 256);
  if (e == hipSuccess && lq_cap > 0) e = hipMemset(h->lq.arrived, 0, (size_t)lq_cap * 4);
  if (e == hipSuccess) e = hipStreamSynchronize(nullptr);
  if (e != hipSuccess) {
    delete h->enqueue;
    free(meta);
    (void)hipFree(dev);
    free(h);
    return EB_ERR_HIP;
  }
  h->h_meta = meta;
  *out = h;
  return EB_OK;
}

eb_status eb_forward(const eb_tables *h, eb_tensor indices, eb_tensor offsets, eb_tensor per_sample_weights,
                     eb_pooling pooling, eb_tensor out) {
  FwdShape sh;
  const eb_status chk = check_forward_args(h, indices, offsets, per_sample_weights, pooling, out, &sh);
  if (chk != EB_OK) return chk;

  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return EB_ERR_HIP;
  if (cur != h->device && hipSetDevice(h->device) != hipSuccess) return EB_ERR_HIP;
  hipError_t e = begin_checked(h);
  if (e == hipSuccess) e = launch_forward(h, indices, offsets, per_sample_weights, pooling, out, sh);
  const eb_status st = end_checked(h, e);
  if (cur != h->device) (void)hipSetDevice(cur);
  return st;
}

eb_status eb_destroy(eb_tables *h) {
  if (!h) return EB_OK;
  int cur = -1;
  eb_status st = EB_OK;
  if (hipGetDevice(&cur) != hipSuccess) st = EB_ERR_HIP;
  if (st == EB_OK && cur != h->device && hipSetDevice(h->device) != hipSuccess) st = EB_ERR_HIP;
  if (st == EB_OK && hipStreamSynchronize(h->stream) != hipSuccess) st = EB_ERR_HIP;
  if (hipFree(h->d_meta) != hipSuccess) st = EB_ERR_HIP;
  free(h->h_meta);
  delete h->enqueue;
  if (cur >= 0 && cur != h->device) (void)hipSetDevice(cur);
  free(h);
  return st;
}

}  // extern "C"
