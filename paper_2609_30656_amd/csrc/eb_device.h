// eb_device.h — internal to libeb: the table descriptor the kernels read, the
// 16-byte-slice row gather with its convert/accumulate step, and the
// cross-lane reduce-scatter, shared by the pooled and un-pooled lookups, the
// FM pass and the backward; and the host-side checks the lookups share.
// Not part of the C ABI (include/eb.h is).
#ifndef EB_DEVICE_H_
#define EB_DEVICE_H_

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>

#include "eb.h"

// Unweighted int8 row-wise pooling sums s*q and the biases separately (one
// fma per element instead of two); 0 keeps the per-element dequantisation.
#ifndef EB_INT8_SPLIT_BIAS
#define EB_INT8_SPLIT_BIAS 1
#endif

namespace eb {

constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kBlock = kWave * kWavesPerBlock;
constexpr int kPassBytes = kWave * 16;  // one wave-wide 16-byte load covers 1 KiB
constexpr uint32_t kBadRow = 0xFFFFFFFFu;
constexpr int kMaxDim = 8192;
// An all-zero row as long as the widest row slice any lane can address
// (8192 fp32 values) plus the int8 scale/bias word.
constexpr size_t kZeroBytes = 4 * kMaxDim + 16;
// A wavefront pools up to this many consecutive bags (their offsets are read
// with one vector load, one per lane, so at most 63).
constexpr int kMaxBagsPerWave = 32;
// Wavefronts resident on a full MI355X (256 CUs x 4 SIMDs x 8 waves).
constexpr int64_t kResidentWaves = 256 * 4 * 8;
constexpr int64_t kTailGens = 4;  // default taper of the lookup's runs (sets of resident wavefronts)
// The backward keeps one gradient row slice per lane: rows of up to 64 lanes
// x 4 fp32 values.
constexpr int kMaxBackwardDim = 256;
// Handles with at most this many tables renumber workgroups XCD-contiguously.
constexpr int32_t kRemapMaxTables = 32;

// Long bags: the lookup leaves bags of more than kDefaultLongBag lookups
// (EB_LONG_BAG at create time) to a second kernel, which pools them in
// segments of up to kLongSegMax positions spread over its workgroups.
constexpr int64_t kDefaultLongBag = 1024;
// Without EB_LONG_BAG the pass runs for batches of at least this many
// lookups, or of at least this many lookups per bag on average.
constexpr int64_t kLongPassMinLookups = (int64_t)1 << 23;
constexpr int64_t kLongPassMinMean = 64;
constexpr int32_t kDefaultLongSeg = 2048;          // positions per segment
constexpr int32_t kLongSegMax = 2048;              // (a segment's indices are staged in LDS)
constexpr int64_t kLqMaxEntries = 16384;           // segments queued per launch
constexpr int64_t kLqMaxPartialFloats = 1 << 24;   // their partial rows: 64 MiB at most
// counter words of LongQueue::ctrl
enum : int { kLqTail = 0, kLqHead = 1, kLqFinished = 2 };

// A handle's queue of long-bag segments (device memory).  Entry e names a
// bag and the bag's first entry; the bag's K segments take K consecutive
// entries, and arrived[first] counts the segments pooled so far.
struct LongQueue {
  uint32_t *ctrl;     // kLqTail: entries reserved; kLqHead: entries taken; kLqFinished: workgroups done
  uint32_t *bag;      // [cap] bag id of each entry
  uint32_t *first;    // [cap] first entry of the entry's bag
  uint32_t *arrived;  // [cap] segments done, per first entry
  float *part;        // [cap][part_ld] each segment's partial sum
  int32_t cap;        // entries (0: no queue, long bags are not split)
  int32_t part_ld;
};

// error bits raised by the kernel, reported in checked mode
constexpr int kErrIndex = 1;
constexpr int kErrOffsets = 2;
constexpr int kErrOutSize = 4;  // an output row would fall outside the output
constexpr int kErrSortWait = 8;  // a sort block gave up waiting for its predecessor's counts

enum : int32_t { kF32 = 0, kF16 = 1, kU8 = 2 };

// Per-table descriptor as the kernel sees it (read through the scalar cache).
struct TableMeta {
  const unsigned char *data;
  int64_t state_base;   // first optimizer-state slot: rows of the earlier tables
  // int8 row-wise tables: row r's 4-byte scale/bias word is at
  // sb_base + r * sb_stride (packed rows: data + dim and the row stride;
  // split layout: the block after all rows' codes, 4 bytes per row)
  const unsigned char *sb_base;
  uint32_t sb_stride;
  uint32_t row_stride;  // bytes
  int32_t num_rows;
  int32_t dim;
  int32_t code_bytes;   // element bytes per row: 4*dim, 2*dim or dim
  int32_t out_col;      // first output column of this table
  int32_t kind;         // dtype * 8 + log2(lanes per row)
  int32_t passes;       // 1 KiB column passes per row
  uint32_t key_base;    // backward sort keys: sum over earlier tables of (rows + 1)
};

// Table rows are plain device memory: address them in the global address
// space so gathers compile to global (not flat) loads.
#define EB_GLOBAL __attribute__((address_space(1)))
typedef const EB_GLOBAL unsigned char gbyte;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
// same vector, only 4-byte aligned: int8 rows of D+4 bytes start on any dword
typedef uint32_t u32x4_a4 __attribute__((ext_vector_type(4), aligned(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int DT>
struct Vals {
  static constexpr int n = DT == kF32 ? 4 : (DT == kF16 ? 8 : 16);  // values per 16 B
  static constexpr int esize = DT == kF32 ? 4 : (DT == kF16 ? 2 : 1);
};

__device__ __forceinline__ float half_lo(uint32_t v) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(v & 0xFFFFu));
}
__device__ __forceinline__ float half_hi(uint32_t v) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(v >> 16));
}

// acc += x (or acc = w*x + acc) for the 16-byte slice v of one row.
//   `one` is 1.0f passed in at run time: fmaf(x, one, acc) with an fp16 x
//   then compiles to a single v_fma_mix_f32 that widens and adds (exact
//   widening, one rounding: the same bits as acc + x).
//   Unweighted int8 rows (SPLIT) accumulate s*q with one fma per element
//   (s*q is exact in fp32) and the row's bias once into cb; the caller adds
//   cb to every element before the cross-lane reduction.  For a one-row bag
//   that gives fp32(s*q + c) exactly as the dequantisation is defined; for
//   longer bags it is a reassociation of the same sum.
template <int DT, bool W, bool SPLIT>
__device__ __forceinline__ void accumulate(float (&acc)[Vals<DT>::n], float &cb, u32x4 v, uint32_t sb, float w,
                                           float one) {
  if constexpr (DT == kF32) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float x = __uint_as_float(v[i]);
      acc[i] = W ? fmaf(w, x, acc[i]) : acc[i] + x;
    }
  } else if constexpr (DT == kF16) {
    const float f = W ? w : one;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc[2 * i] = fmaf(half_lo(v[i]), f, acc[2 * i]);
      acc[2 * i + 1] = fmaf(half_hi(v[i]), f, acc[2 * i + 1]);
    }
  } else if constexpr (SPLIT && !W) {
    const float s = half_lo(sb);
    cb = fmaf(half_hi(sb), one, cb);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[4 * i + j] = fmaf(s, (float)((v[i] >> (8 * j)) & 0xFFu), acc[4 * i + j]);
    }
  } else {
    // x = fp32(s*q + c): s*q is exact in fp32 (11-bit by 8-bit significands),
    // so the fma rounds once, as the dequantisation is defined
    const float s = half_lo(sb), c = half_hi(sb);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float q = (float)((v[i] >> (8 * j)) & 0xFFu);
        const float x = fmaf(s, q, c);
        acc[4 * i + j] = W ? fmaf(w, x, acc[4 * i + j]) : acc[4 * i + j] + x;
      }
    }
  }
}

// Row `row`'s scale/bias word of an int8 row-wise table (see TableMeta).
__device__ __forceinline__ gbyte *sb_word(const TableMeta &m, uint32_t row) {
  return (gbyte *)m.sb_base + (uint64_t)row * m.sb_stride;
}

template <int DT>
__device__ __forceinline__ u32x4 load_slice(gbyte *p) {
  if constexpr (DT == kU8) {
    return *reinterpret_cast<const EB_GLOBAL u32x4_a4 *>(p);
  } else {
    return *reinterpret_cast<const EB_GLOBAL u32x4 *>(p);
  }
}

// Row-load steps issued before the first is consumed: enough rows in flight
// per wave to cover HBM latency within the register budget.
#ifndef EB_INT8_MAX_UNROLL
#define EB_INT8_MAX_UNROLL 4
#endif
#ifndef EB_WEIGHTED_MAX_UNROLL
#define EB_WEIGHTED_MAX_UNROLL 4
#endif
template <int DT, int RPL, bool W>
struct Unroll {
  static constexpr int c0 = DT == kU8 ? EB_INT8_MAX_UNROLL : 8;
  static constexpr int cap = W && EB_WEIGHTED_MAX_UNROLL < c0 ? EB_WEIGHTED_MAX_UNROLL : c0;
  static constexpr int u = (kWave / RPL) < cap ? (kWave / RPL) : cap;
};

// Steps per batch of the pooled gather: as Unroll, except that fp16 rows of
// 128 bytes (8 rows per load) take batches of 4 steps (32 rows).  With 8, the
// kernel that switches over every fp16 width needs 66 VGPRs (7 waves per
// SIMD); with 4 it fits in 64 (8 waves), 2% faster on a mixed-width workload.
template <int DT, int RPL, bool W>
struct GatherUnroll {
  static constexpr int u = (DT == kF16 && RPL == 8 && Unroll<DT, RPL, W>::u > 4) ? 4 : Unroll<DT, RPL, W>::u;
};

// 64-bit value of lane `l` (wave-uniform l) of a per-lane value.
__device__ __forceinline__ int64_t readlane64(int64_t v, int l) {
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, l);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)((uint64_t)v >> 32), l);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// What the row gather needs besides the table: the all-zero row read in
// place of rows that do not exist, 1.0f as a run-time value, and the word
// that records an index outside its table.
struct GatherCtx {
  const unsigned char *zero;  // kZeroBytes of zeros
  int *err;
  float one;
};

// One chunk of up to 64 consecutive index positions of a bag, one per lane,
// as the gathers use it.
struct Chunk {
  uint32_t row;  // row number, or kBadRow (no row / outside the table)
  float w;       // per-sample weight (weighted pooling only; 0 past the chunk)
  int n;         // positions in the chunk (wave-uniform)
};

// The same chunk as read: each lane's index bits (hi only for 64-bit indices)
// and weight, with the loads possibly still in flight.  resolve() makes the
// Chunk where it is used, so a chunk loaded ahead stays in flight until then
// (checking an index right after its load would make the wave wait for it
// before the current chunk's rows are even requested).
struct RawChunk {
  uint32_t lo, hi;
  float w;
  int n;
};

// Positions [c, min(c + 64, end)) of the index stream, one per lane, with
// their weights.  Lanes past the chunk re-read its first position, so no
// branch surrounds the loads.  Indices and weights are read once, so they
// are streamed past the caches.
template <bool W>
__device__ __forceinline__ RawChunk load_chunk(const void *indices, const float *weights, int idx64, int64_t c,
                                               int64_t end) {
  const int lane = threadIdx.x & (kWave - 1);
  RawChunk k;
  k.n = (int)((end - c) < kWave ? (end - c) : kWave);
  k.lo = 0u;
  k.hi = 0u;
  k.w = 0.0f;
  if (k.n > 0) {
    const int64_t p = c + (lane < k.n ? lane : 0);
    if (idx64) {
      const uint64_t v = __builtin_nontemporal_load(static_cast<const uint64_t *>(indices) + p);
      k.lo = (uint32_t)v;
      k.hi = (uint32_t)(v >> 32);
    } else {
      k.lo = __builtin_nontemporal_load(static_cast<const uint32_t *>(indices) + p);
    }
    if constexpr (W) k.w = __builtin_nontemporal_load(weights + p);
  }
  return k;
}

// The rows of a chunk of a table of num_rows rows: an index outside
// [0, num_rows) and a lane past the chunk give kBadRow (and weight 0).
__device__ __forceinline__ Chunk resolve(const RawChunk &k, int32_t num_rows, int idx64) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t r = idx64 ? (int64_t)(((uint64_t)k.hi << 32) | k.lo) : (int64_t)(int32_t)k.lo;
  Chunk c;
  c.n = k.n;
  c.row = (lane < k.n && r >= 0 && r < num_rows) ? (uint32_t)r : kBadRow;
  c.w = lane < k.n ? k.w : 0.0f;
  return c;
}

// Store KEEP consecutive pooled values (16-, 8- or 4-byte non-temporal stores:
// the output is written once and not read back by the lookup).
template <int KEEP>
__device__ __forceinline__ void store_slice(float *dst, const float (&v)[KEEP]) {
  if constexpr (KEEP % 4 == 0) {
#pragma unroll
    for (int i = 0; i < KEEP; i += 4)
      __builtin_nontemporal_store(f32x4{v[i], v[i + 1], v[i + 2], v[i + 3]}, reinterpret_cast<f32x4 *>(dst + i));
  } else if constexpr (KEEP == 2) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    __builtin_nontemporal_store(f32x2{v[0], v[1]}, reinterpret_cast<f32x2 *>(dst));
  } else {
    __builtin_nontemporal_store(v[0], dst);
  }
}

// Gather steps [s0, s0 + N) of one chunk (RPL rows per step) and add them into
// this lane's accumulators.  Straight-line code: a lane whose row does not
// exist (past the chunk's end, outside the table, or a slice past the row's
// end) reads the handle's all-zero row instead, which adds nothing, so no
// branch separates a load from its use and the loads of all N steps are in
// flight together.
template <int DT, int LPR, bool W, bool SPLIT, int N>
__device__ __forceinline__ void gather_steps(const TableMeta &m, const GatherCtx &a, const Chunk &k, int s0,
                                             float (&acc)[Vals<DT>::n], float &cb, int colb, bool colok,
                                             int base = 0) {
  constexpr int RPL = kWave / LPR;
  const int lane = threadIdx.x & (kWave - 1);
  const int grp = lane / LPR;
  u32x4 v[N];
  uint32_t sb[N];
  float w[N];
#pragma unroll
  for (int u = 0; u < N; ++u) {
    const int r = (s0 + u) * RPL + grp;  // entry of the range [base, base + k.n)
    uint32_t row;
    if constexpr (RPL == 1) {
      row = __builtin_amdgcn_readlane(k.row, (base + s0 + u) & (kWave - 1));
      if constexpr (W)
        w[u] = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(uint32_t, k.w),
                                                                    (base + s0 + u) & (kWave - 1)));
    } else {
      row = (uint32_t)__shfl((int)k.row, (base + r) & (kWave - 1));
      if constexpr (W) w[u] = __shfl(k.w, (base + r) & (kWave - 1));
    }
    const bool ok = (r < k.n) && (row != kBadRow) && colok;
    gbyte *p = ok ? (gbyte *)m.data + (uint64_t)row * m.row_stride : (gbyte *)a.zero;
    v[u] = load_slice<DT>(p + colb);
    if constexpr (DT == kU8) sb[u] = *reinterpret_cast<const EB_GLOBAL uint32_t *>(ok ? sb_word(m, row) : p);
    else sb[u] = 0u;
    if constexpr (!W) w[u] = 1.0f;
  }
#pragma unroll
  for (int u = 0; u < N; ++u) accumulate<DT, W, SPLIT>(acc, cb, v[u], sb[u], w[u], a.one);
}

// One straight-line batch of exactly `rem` steps (1 <= rem <= N).
template <int DT, int LPR, bool W, bool SPLIT, int N>
__device__ __forceinline__ void gather_exact(int rem, const TableMeta &m, const GatherCtx &a, const Chunk &k, int s,
                                             float (&acc)[Vals<DT>::n], float &cb, int colb, bool colok) {
  if constexpr (N > 0) {
    if (rem == N) {
      gather_steps<DT, LPR, W, SPLIT, N>(m, a, k, s, acc, cb, colb, colok);
      return;
    }
    gather_exact<DT, LPR, W, SPLIT, N - 1>(rem, m, a, k, s, acc, cb, colb, colok);
  }
}

// Gather all rows of one chunk: full batches of U steps, then one batch for
// the rest, so a chunk of up to U steps costs one memory round trip.  With
// batches of 8 the last one has exactly the remaining steps: padding it to a
// power of two spent up to 3 of every 8 loads on the zero row (a 20-row bag
// of 4 rows per load takes 5 steps), which cost 7% on 26 fp32 D64 tables at
// batch 2048 with Poisson(20) bags.  With batches of 4 it
// is padded to 2 or 4 steps (at most one padded load): exact sizes there were
// no faster and took more registers.
template <int DT, int LPR, bool W, bool SPLIT>
__device__ __forceinline__ void gather_chunk(const TableMeta &m, const GatherCtx &a, const Chunk &k,
                                             float (&acc)[Vals<DT>::n], float &cb, int colb, bool colok) {
  constexpr int RPL = kWave / LPR;
  constexpr int U = GatherUnroll<DT, RPL, W>::u;
  const int lane = threadIdx.x & (kWave - 1);
  if (__ballot(lane < k.n && k.row == kBadRow)) {
    if (lane == 0) atomicOr(a.err, kErrIndex);
  }
  const int steps = (k.n + RPL - 1) / RPL;
  int s = 0;
  if constexpr (U >= 8) {
    for (; steps - s >= U; s += U) gather_steps<DT, LPR, W, SPLIT, U>(m, a, k, s, acc, cb, colb, colok);
    if (steps > s) gather_exact<DT, LPR, W, SPLIT, U - 1>(steps - s, m, a, k, s, acc, cb, colb, colok);
  } else {
    for (; steps - s > U / 2; s += U) gather_steps<DT, LPR, W, SPLIT, U>(m, a, k, s, acc, cb, colb, colok);
    const int rem = steps - s;  // 0 .. U/2
    if constexpr (U >= 4) {
      if (rem > 1) {
        gather_steps<DT, LPR, W, SPLIT, 2>(m, a, k, s, acc, cb, colb, colok);
        return;
      }
    }
    if (rem > 0) gather_steps<DT, LPR, W, SPLIT, 1>(m, a, k, s, acc, cb, colb, colok);
  }
}

// One straight-line batch of exactly `rem` steps of entries from `base` on.
template <int DT, int LPR, bool W, int N>
__device__ __forceinline__ void gather_exact_at(int rem, const TableMeta &m, const GatherCtx &a, const Chunk &k, int s,
                                                float (&acc)[Vals<DT>::n], float &cb, int colb, bool colok,
                                                int base) {
  if constexpr (N > 0) {
    if (rem == N) {
      gather_steps<DT, LPR, W, false, N>(m, a, k, s, acc, cb, colb, colok, base);
      return;
    }
    gather_exact_at<DT, LPR, W, N - 1>(rem, m, a, k, s, acc, cb, colb, colok, base);
  }
}

// Gather entries [base, base + n) of a chunk (n <= 64 - base) and accumulate
// them: the same batching as gather_chunk, for a run that covers only part
// of the chunk.
template <int DT, int LPR, bool W>
__device__ __forceinline__ void gather_range(const TableMeta &m, const GatherCtx &a, Chunk k, int base, int n,
                                             float (&acc)[Vals<DT>::n], int colb, bool colok) {
  constexpr int RPL = kWave / LPR;
  constexpr int U = GatherUnroll<DT, RPL, W>::u;
  float cb = 0.0f;
  k.n = n;
  const int steps = (n + RPL - 1) / RPL;
  int s = 0;
  if constexpr (U >= 8) {
    for (; steps - s >= U; s += U) gather_steps<DT, LPR, W, false, U>(m, a, k, s, acc, cb, colb, colok, base);
    if (steps > s) gather_exact_at<DT, LPR, W, U - 1>(steps - s, m, a, k, s, acc, cb, colb, colok, base);
    return;
  }
  for (; steps - s > U / 2; s += U) gather_steps<DT, LPR, W, false, U>(m, a, k, s, acc, cb, colb, colok, base);
  const int rem = steps - s;
  if constexpr (U >= 8) {
    if (rem > 2) {
      gather_steps<DT, LPR, W, false, 4>(m, a, k, s, acc, cb, colb, colok, base);
      return;
    }
  }
  if constexpr (U >= 4) {
    if (rem > 1) {
      gather_steps<DT, LPR, W, false, 2>(m, a, k, s, acc, cb, colb, colok, base);
      return;
    }
  }
  if (rem > 0) gather_steps<DT, LPR, W, false, 1>(m, a, k, s, acc, cb, colb, colok, base);
}

__device__ __forceinline__ float dpp_row_ror(float x, int o) {
  // rotate within each 16-lane row by o lanes (o is a compile-time constant)
  const int xi = __builtin_bit_cast(int, x);
  int r;
  switch (o) {
    case 1: r = __builtin_amdgcn_update_dpp(0, xi, 0x121, 0xf, 0xf, false); break;
    case 2: r = __builtin_amdgcn_update_dpp(0, xi, 0x122, 0xf, 0xf, false); break;
    case 4: r = __builtin_amdgcn_update_dpp(0, xi, 0x124, 0xf, 0xf, false); break;
    default: r = __builtin_amdgcn_update_dpp(0, xi, 0x128, 0xf, 0xf, false); break;
  }
  return __builtin_bit_cast(float, r);
}

// Sum the RPL row groups' partial vectors (a reduce-scatter in a fixed order,
// so results are deterministic).  On return, lane (row q of 16 lanes, slot
// p) holds V / min(RPL, 4) consecutive values of the pooled slice of lane-slot
// p % LPR, starting at value index first_value(); only lanes with
// stores() == true write them.
// (Elements of the swap builtins' two-lane result are read by value with
// __uint_as_float: __builtin_bit_cast applied to such an element reads the
// first element whatever the index.)
template <int DT, int LPR>
struct Reduce {
  static constexpr int V = Vals<DT>::n;
  static constexpr int KEEP = LPR >= 64 ? V : (LPR == 32 ? V / 2 : V / 4);

  __device__ static __forceinline__ void run(float (&acc)[V]) {
    if constexpr (LPR < 16) {
      // combine the row groups that share a 16-lane row: all-reduce by rotation
#pragma unroll
      for (int o = LPR; o < 16; o <<= 1) {
#pragma unroll
        for (int i = 0; i < V; ++i) acc[i] += dpp_row_ror(acc[i], o);
      }
    }
    if constexpr (LPR <= 16) {
      // rows 0+1 and 2+3: pair value i with value i + V/2; rows 0,2 keep the
      // first, rows 1,3 the second
#pragma unroll
      for (int i = 0; i < V / 2; ++i) {
        const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(acc[i]),
                                                        __float_as_uint(acc[i + V / 2]), false, false);
        acc[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
      }
      // halves: pair value j with j + V/4 (of the V/2 left); the low half
      // keeps the first, the high half the second
#pragma unroll
      for (int j = 0; j < V / 4; ++j) {
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[j]),
                                                        __float_as_uint(acc[j + V / 4]), false, false);
        acc[j] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
      }
    } else if constexpr (LPR == 32) {
#pragma unroll
      for (int i = 0; i < V / 2; ++i) {
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[i]),
                                                        __float_as_uint(acc[i + V / 2]), false, false);
        acc[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
      }
    }
  }

  // index (within the lane-slot's V values) of the first value this lane holds
  __device__ static __forceinline__ int first_value(int lane) {
    if constexpr (LPR >= 64) {
      return 0;
    } else if constexpr (LPR == 32) {
      return (lane >> 5) * (V / 2);
    } else {
      const int q = lane >> 4;  // 16-lane row
      return ((q & 1) ? V / 2 : 0) + ((q & 2) ? V / 4 : 0);
    }
  }

  __device__ static __forceinline__ bool stores(int lane) {
    if constexpr (LPR >= 16) return true;
    return (lane & 15) < LPR;
  }
};

// Workgroups are handed to the 8 XCDs round-robin (block i runs on XCD i % 8).
// Renumbering them so each XCD walks one contiguous eighth of the work keeps
// each XCD's L2 on few tables for the whole launch; leaving them round-robin
// puts all XCDs on the same table at once, so the shared Infinity Cache holds
// that one table's hot rows.  The first wins with few tables (measured: 8 and
// 26), the second with many large ones (64 and 100); the host picks.
__device__ __forceinline__ uint32_t xcd_contiguous(uint32_t i, uint32_t n) {
  constexpr uint32_t kXcd = 8;
  const uint32_t x = i % kXcd, slot = i / kXcd;
  const uint32_t q = n / kXcd, r = n % kXcd;
  return x < r ? x * (q + 1) + slot : r * (q + 1) + (x - r) * q + slot;
}

__host__ __device__ inline int log2_lanes_per_row(int code_bytes) {
  int slices = (code_bytes + 15) / 16;
  int l = 0;
  while ((1 << l) < slices && l < 6) ++l;
  return l;
}

// Host side, shared by the entry points that pool (defined in eb_forward.hip;
// hidden: the library exports only the C ABI).
#define EB_INTERNAL __attribute__((visibility("hidden")))
struct FwdShape {
  int64_t num_bags;
  int64_t batch;
  bool weighted;
};
// The argument checks of eb_forward (every host-detectable error, before
// anything is enqueued).
EB_INTERNAL eb_status check_forward_args(const struct ::eb_tables *h, const eb_tensor &indices, const eb_tensor &offsets,
                             const eb_tensor &weights, eb_pooling pooling, const eb_tensor &out, FwdShape *sh);
// Enqueue the pooled lookup (arguments already checked).
EB_INTERNAL hipError_t launch_forward(const struct ::eb_tables *h, const eb_tensor &indices, const eb_tensor &offsets,
                                      const eb_tensor &weights, eb_pooling pooling, const eb_tensor &out,
                                      const FwdShape &sh);
// Checked mode: clear the device error word before the launches, then read it
// back (after a stream sync) and turn it into a status.
EB_INTERNAL hipError_t begin_checked(const struct ::eb_tables *h);
EB_INTERNAL eb_status end_checked(const struct ::eb_tables *h, hipError_t e);

}  // namespace eb

struct eb_tables {
  int device;
  hipStream_t stream;
  int32_t num_tables;
  int32_t checked;
  int32_t bags_per_wave;  // 0: chosen per call from the bag count
  int64_t tail_bags;      // lookup taper: bags per table in short runs at the end (-1: chosen per call)
  int32_t tail_run;       // bags per such run
  int64_t long_bag_len;   // > 0: bags with more lookups go to the long-bag pass (0: none do)
  int32_t long_bag_forced;  // EB_LONG_BAG set: the pass runs for batches of any size
  int32_t long_seg_log2;  // that pass pools them in segments of 2^long_seg_log2 positions
  eb::LongQueue lq;       // its queue (inside the d_meta allocation)
  // A lookup launch and its long-bag pass follow each other on the stream
  // (the pass takes what the launch queued): calls from several host threads
  // enqueue them under this lock.
  std::mutex *enqueue;
  int32_t dtype_mask;     // bit d set: some table has storage type d
  int32_t single_log2;    // lanes-per-row log2 shared by every table of one type, else -1
  int32_t xcd_remap;      // see xcd_contiguous
  int64_t sum_dim;
  int32_t backward_ok;    // every table fp32/fp16 with dim <= 256, sort keys fit in 32 bits
  int32_t bwd_tile_chunks;  // 0: chosen per call; else backward tiles of this many 64-position chunks
  int32_t bwd_sort_items;   // 0: chosen per call; else 4, 8, 12 or 16 elements per thread of the backward's sort
  int32_t bwd_xcd_remap;    // backward tiles in XCD-contiguous order
  int32_t max_dim;
  int32_t uniform_dim;    // the dim every table shares, or 0 if they differ
  int64_t total_rows;     // sum of the tables' row counts (optimizer-state length)
  eb::TableMeta *d_meta;  // device: descriptors, then the error word, then the zero row
  eb::TableMeta *h_meta;  // host copy of the descriptors
  int *d_err;
  unsigned char *d_zero;
};


#endif  // EB_DEVICE_H_
