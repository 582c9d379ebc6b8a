// libeb — un-pooled (sequence) lookup.
//
// Sequence recommenders (the paper's Introduction names HSTU among the
// architectures its profiling targets) consume the embedding of every
// position of a jagged feature instead of a pooled sum.  For table t and
// every position i in [start_t, end_t) = [offsets[t*B], offsets[(t+1)*B]):
//
//   out[base_t + (i - start_t) * D_t + d] = x(t, idx[i], d),   base_t = sum_{s<t} N_s D_s
//
// so table t's positions form a [N_t, D_t] block and the blocks follow in
// table order ([N, D] when all tables share D).  x is the fp32 element value
// of the pooled lookup: each is one exact conversion (or one rounding for
// int8 row-wise rows), so the output matches its definition bit for bit.
//
// Work map: a wavefront takes a span of 64*k consecutive positions.  It finds
// the table of its first position once (the lanes test 64 tables' start
// offsets at a time and sum the earlier tables' output sizes), then walks the
// span as a stream of chunks of up to 64 positions inside one table, loading
// the next chunk's indices before the current chunk's rows are gathered.
// Rows are gathered as in the pooled lookup (LPR lanes per row, RPL rows per
// wave-wide load, straight-line batches), converted, and stored with
// non-temporal 16-byte stores that fill whole lines (see Piece); every store
// is checked against the output's size.  The bag offsets inside a table are not read: only the T+1 table
// starts offsets[t*B] matter here.

#include "eb_device.h"

namespace eb {
namespace {

struct SeqArgs {
  const TableMeta *meta;
  GatherCtx ctx;
  const void *indices;
  const void *offsets;
  float *out;
  int64_t num_indices;
  int64_t out_numel;
  int64_t num_waves;
  int32_t batch;
  int32_t num_tables;
  int32_t idx64;
  int32_t span;  // positions per wavefront, a multiple of 64
};

// offsets[t*B] clamped into [0, N]; *bad is set if it was outside
__device__ __forceinline__ int64_t table_start(const SeqArgs &a, int32_t t, bool *bad) {
  const int64_t g = (int64_t)t * a.batch;
  const int64_t v = a.idx64 ? static_cast<const int64_t *>(a.offsets)[g]
                            : (int64_t) static_cast<const int32_t *>(a.offsets)[g];
  if (v < 0 || v > a.num_indices) {
    *bad = true;
    return v < 0 ? 0 : a.num_indices;
  }
  return v;
}

__device__ __forceinline__ int64_t wave_sum64(int64_t v) {
#pragma unroll
  for (int o = kWave / 2; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// A lane's share of a row in a column window (16 bytes) is read as P pieces
// of PB bytes, piece j of lane slot s at byte col + PB*(s + LPR*j), each
// converted to F = PB / element-size fp32 values, so store j of the LPR lanes
// of a row writes one contiguous run.  Measured on MI355X with non-temporal
// stores: int8 rows read as 16-byte pieces (each lane's stores covering 16 of
// every 64 bytes) ran 3x slower than as 8-byte pieces (16 of every 32); fp16
// rows are fastest as 16-byte pieces (16 of every 32 bytes), fp32 rows write
// whole runs either way; ordinary stores were slower in every case.
#ifndef EB_SEQ_PB_F16
#define EB_SEQ_PB_F16 16
#endif
#ifndef EB_SEQ_PB_U8
#define EB_SEQ_PB_U8 8
#endif
#ifndef EB_SEQ_NT_STORES
#define EB_SEQ_NT_STORES 1
#endif
template <int DT>
struct Piece {
  static constexpr int bytes = DT == kF32 ? 16 : (DT == kF16 ? EB_SEQ_PB_F16 : EB_SEQ_PB_U8);
  static constexpr int count = 16 / bytes;
  static constexpr int floats = bytes / Vals<DT>::esize;
};

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ void store4(float *dst, float a, float b, float c, float d) {
  if constexpr (EB_SEQ_NT_STORES) __builtin_nontemporal_store(f32x4{a, b, c, d}, reinterpret_cast<f32x4 *>(dst));
  else *reinterpret_cast<f32x4 *>(dst) = f32x4{a, b, c, d};
}

// Write the N steps' converted rows of chunk k (positions [c, c + k.n) of a
// table whose block starts at output element rowbase for position c); col is
// the window's first byte.
template <int DT, int LPR, int N>
__device__ __forceinline__ void copy_steps(const SeqArgs &a, const TableMeta &m, const Chunk &k, int s0, int col,
                                           int64_t rowbase) {
  constexpr int RPL = kWave / LPR;
  constexpr int PB = Piece<DT>::bytes;
  constexpr int P = Piece<DT>::count;
  constexpr int F = Piece<DT>::floats;
  constexpr int W = PB / 4;  // dwords per piece
  const int lane = threadIdx.x & (kWave - 1);
  const int grp = lane / LPR;
  const int slot = lane % LPR;
  u32x4 v[N];
  uint32_t sb[N];
#pragma unroll
  for (int u = 0; u < N; ++u) {
    const int r = (s0 + u) * RPL + grp;
    const uint32_t row = RPL == 1 ? __builtin_amdgcn_readlane(k.row, (s0 + u) & (kWave - 1))
                                  : (uint32_t)__shfl((int)k.row, r & (kWave - 1));
    const bool ok = (r < k.n) && (row != kBadRow);
    gbyte *p = ok ? (gbyte *)m.data + (uint64_t)row * m.row_stride : (gbyte *)a.ctx.zero;
    // a piece past the row's end reads the zero row: no branch separates a
    // load from its use, so the batch's loads stay in flight together
#pragma unroll
    for (int j = 0; j < P; ++j) {
      const int b = col + PB * (slot + LPR * j);
      gbyte *q = b < m.code_bytes ? p + b : (gbyte *)a.ctx.zero;
      if constexpr (W == 4) {
        v[u] = DT == kU8 ? *reinterpret_cast<const EB_GLOBAL u32x4_a4 *>(q)
                         : *reinterpret_cast<const EB_GLOBAL u32x4 *>(q);
      } else if constexpr (W == 2) {
        const u32x2 w = *reinterpret_cast<const EB_GLOBAL u32x2 *>(q);
        v[u][2 * j] = w[0];
        v[u][2 * j + 1] = w[1];
      } else {
        v[u][j] = *reinterpret_cast<const EB_GLOBAL uint32_t *>(q);
      }
    }
    if constexpr (DT == kU8) sb[u] = *reinterpret_cast<const EB_GLOBAL uint32_t *>(ok ? sb_word(m, row) : p);
    else sb[u] = 0u;
  }
#pragma unroll
  for (int u = 0; u < N; ++u) {
    const int r = (s0 + u) * RPL + grp;
    if (r >= k.n) continue;
    const int64_t orow = rowbase + (int64_t)r * m.dim;
#pragma unroll
    for (int j = 0; j < P; ++j) {
      const int b = col + PB * (slot + LPR * j);
      if (b >= m.code_bytes) continue;
      float x[F];
      if constexpr (DT == kF32) {
#pragma unroll
        for (int i = 0; i < 4; ++i) x[i] = __uint_as_float(v[u][i]);
      } else if constexpr (DT == kF16) {
#pragma unroll
        for (int i = 0; i < W; ++i) {
          x[2 * i] = half_lo(v[u][W * j + i]);
          x[2 * i + 1] = half_hi(v[u][W * j + i]);
        }
      } else {
        // fp32(s*q + c), rounded once, as the dequantisation is defined
        const float sc = half_lo(sb[u]), c = half_hi(sb[u]);
#pragma unroll
        for (int i = 0; i < F; ++i) x[i] = fmaf(sc, (float)((v[u][W * j + i / 4] >> (8 * (i % 4))) & 0xFFu), c);
      }
      const int64_t e = orow + b / Vals<DT>::esize;
      if (e + F > a.out_numel) {
        atomicOr(a.ctx.err, kErrOutSize);
        continue;
      }
#pragma unroll
      for (int i = 0; i < F; i += 4) store4(a.out + e + i, x[i], x[i + 1], x[i + 2], x[i + 3]);
    }
  }
}

// All rows of one chunk, in straight-line batches of up to U steps.
template <int DT, int LPR>
__device__ __forceinline__ void copy_chunk(const SeqArgs &a, const TableMeta &m, const Chunk &k, int64_t rowbase) {
  constexpr int RPL = kWave / LPR;
  constexpr int U = Unroll<DT, RPL, false>::u;
  const int lane = threadIdx.x & (kWave - 1);
  if (__ballot(lane < k.n && k.row == kBadRow)) {
    if (lane == 0) atomicOr(a.ctx.err, kErrIndex);
  }
  const int steps = (k.n + RPL - 1) / RPL;
  for (int p = 0; p < m.passes; ++p) {
    const int col = p * kPassBytes;
    int s = 0;
    for (; steps - s > U / 2; s += U) copy_steps<DT, LPR, U>(a, m, k, s, col, rowbase);
    const int rem = steps - s;
    if constexpr (U >= 8) {
      if (rem > 2) {
        copy_steps<DT, LPR, 4>(a, m, k, s, col, rowbase);
        continue;
      }
    }
    if constexpr (U >= 4) {
      if (rem > 1) {
        copy_steps<DT, LPR, 2>(a, m, k, s, col, rowbase);
        continue;
      }
    }
    if (rem > 0) copy_steps<DT, LPR, 1>(a, m, k, s, col, rowbase);
  }
}

#define EB_SEQ_LPR(LOG2)                                  \
  case LOG2:                                              \
    copy_chunk<DT, (1 << (LOG2))>(a, m, ck, rowbase);     \
    break;

// DT: the storage type this launch serves (chunks of other tables are
// walked past).  LOG2 >= 0 fixes the lanes per row; LOG2 < 0 switches on each
// table's.
template <int DT, int LOG2>
__global__ __launch_bounds__(kBlock) void eb_seq_kernel(SeqArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wid = (int64_t)blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  if (wid >= a.num_waves) return;
  const int64_t p0 = wid * a.span;
  const int64_t p1 = (p0 + a.span) < a.num_indices ? (p0 + a.span) : a.num_indices;

  // the table holding p0, its position range, and the first output element of
  // its block (the sizes of the blocks of the tables before it)
  bool bad = false;
  int32_t t = -1;
  int64_t st = 0, en = 0, base = 0;
  for (int32_t g = 0; g < a.num_tables && t < 0; g += kWave) {
    const int32_t l = g + lane;
    int64_t s0 = 0, s1 = 0, before = 0;
    bool mine = false;
    if (l < a.num_tables) {
      s0 = table_start(a, l, &bad);
      s1 = table_start(a, l + 1, &bad);
      if (s1 < s0) {
        bad = true;
        s1 = s0;
      }
      mine = s0 <= p0 && p0 < s1;
      if (s1 <= p0) before = (s1 - s0) * a.meta[l].dim;
    }
    base += wave_sum64(before);
    const uint64_t hit = __ballot(mine);
    if (hit) {
      const int j = __builtin_ctzll(hit);
      t = g + j;
      st = readlane64(s0, j);
      en = readlane64(s1, j);
    }
  }
  if (__ballot(bad) && lane == 0) atomicOr(a.ctx.err, kErrOffsets);
  if (t < 0) {
    if (lane == 0) atomicOr(a.ctx.err, kErrOffsets);  // offsets do not cover this position
    return;
  }

  TableMeta m = a.meta[t];
  int64_t c = p0;
  int64_t hi = en < p1 ? en : p1;
  hi = (c + kWave) < hi ? (c + kWave) : hi;
  RawChunk cur = load_chunk<false>(a.indices, nullptr, a.idx64, c, hi);
  while (true) {
    // the next chunk: the rest of this table's part of the span, or the next
    // non-empty table's first positions
    int64_t cn = hi;
    int32_t tn = t;
    int64_t stn = st, enn = en, basen = base;
    bool more = cn < p1;
    if (more && cn >= en) {
      bool badn = false;
      while (cn >= enn && tn + 1 < a.num_tables) {
        basen += (enn - stn) * a.meta[tn].dim;
        ++tn;
        stn = enn;
        int64_t e2 = table_start(a, tn + 1, &badn);
        enn = e2 < stn ? stn : e2;
        if (e2 < stn) badn = true;
      }
      if (badn && lane == 0) atomicOr(a.ctx.err, kErrOffsets);
      if (cn >= enn || cn != stn) {  // positions past the last table, or a gap
        if (lane == 0) atomicOr(a.ctx.err, kErrOffsets);
        more = false;
      }
    }
    int64_t hin = 0;
    RawChunk nxt;
    if (more) {
      hin = enn < p1 ? enn : p1;
      hin = (cn + kWave) < hin ? (cn + kWave) : hin;
      nxt = load_chunk<false>(a.indices, nullptr, a.idx64, cn, hin);
    }

    if (m.kind / 8 == DT) {
      const int64_t rowbase = base + (c - st) * m.dim;
      const Chunk ck = resolve(cur, m.num_rows, a.idx64);
      if constexpr (LOG2 >= 0) {
        copy_chunk<DT, (1 << (LOG2 >= 0 ? LOG2 : 0))>(a, m, ck, rowbase);
      } else {
        switch (m.kind % 8) {
          EB_SEQ_LPR(0) EB_SEQ_LPR(1) EB_SEQ_LPR(2) EB_SEQ_LPR(3) EB_SEQ_LPR(4) EB_SEQ_LPR(5) EB_SEQ_LPR(6)
          default:
            break;
        }
      }
    }
    if (!more) break;
    if (tn != t) m = a.meta[tn];
    t = tn;
    st = stn;
    en = enn;
    base = basen;
    c = cn;
    hi = hin;
    cur = nxt;
  }
}

#undef EB_SEQ_LPR

typedef void (*SeqKernelFn)(SeqArgs);

template <int DT>
SeqKernelFn pick_seq(int log2) {
  switch (log2) {
    case 0: return eb_seq_kernel<DT, 0>;
    case 1: return eb_seq_kernel<DT, 1>;
    case 2: return eb_seq_kernel<DT, 2>;
    case 3: return eb_seq_kernel<DT, 3>;
    case 4: return eb_seq_kernel<DT, 4>;
    case 5: return eb_seq_kernel<DT, 5>;
    case 6: return eb_seq_kernel<DT, 6>;
    default: return eb_seq_kernel<DT, -1>;
  }
}

SeqKernelFn pick_seq(int dt, int log2) {
  if (dt == kF32) return pick_seq<kF32>(log2);
  if (dt == kF16) return pick_seq<kF16>(log2);
  return pick_seq<kU8>(log2);
}

}  // namespace
}  // namespace eb

using namespace eb;

extern "C" eb_status eb_forward_seq(const eb_tables *h, eb_tensor indices, eb_tensor offsets, eb_tensor out) {
  if (!h) return EB_ERR_INVALID_ARG;
  if (indices.elem_type != EB_I32 && indices.elem_type != EB_I64) return EB_ERR_DTYPE;
  if (offsets.elem_type != indices.elem_type) return EB_ERR_DTYPE;
  if (out.elem_type != EB_T_F32) return EB_ERR_DTYPE;
  if (!offsets.data) return EB_ERR_INVALID_ARG;
  if (indices.numel < 0 || (indices.numel > 0 && !indices.data)) return EB_ERR_INVALID_ARG;
  if (out.numel < 0 || (out.numel > 0 && !out.data)) return EB_ERR_INVALID_ARG;
  if (offsets.numel < 2 || (offsets.numel - 1) % h->num_tables != 0) return EB_ERR_SHAPE;
  const int64_t batch = (offsets.numel - 1) / h->num_tables;
  if (offsets.numel - 1 > INT32_MAX) return EB_ERR_SHAPE;
  const int64_t n = indices.numel;
  // each position writes one row of its table's width
  int32_t min_dim = h->max_dim;
  for (int32_t t = 0; t < h->num_tables; ++t)
    if (h->h_meta[t].dim < min_dim) min_dim = h->h_meta[t].dim;
  if (h->uniform_dim ? out.numel != n * h->uniform_dim : (out.numel < n * min_dim || out.numel > n * h->max_dim))
    return EB_ERR_SHAPE;
  const size_t isz = indices.elem_type == EB_I64 ? 8 : 4;
  if (reinterpret_cast<uintptr_t>(out.data) % 16 != 0 || reinterpret_cast<uintptr_t>(offsets.data) % isz != 0 ||
      reinterpret_cast<uintptr_t>(indices.data) % isz != 0)
    return EB_ERR_UNSUPPORTED;
  if (n == 0) return EB_OK;

  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return EB_ERR_HIP;
  if (cur != h->device && hipSetDevice(h->device) != hipSuccess) return EB_ERR_HIP;

  SeqArgs a;
  a.meta = h->d_meta;
  a.ctx.err = h->d_err;
  a.ctx.zero = h->d_zero;
  a.ctx.one = 1.0f;
  a.indices = indices.data;
  a.offsets = offsets.data;
  a.out = static_cast<float *>(const_cast<void *>(out.data));
  a.num_indices = n;
  a.out_numel = out.numel;
  a.batch = (int32_t)batch;
  a.num_tables = h->num_tables;
  a.idx64 = indices.elem_type == EB_I64;
  // chunks of 64 positions per wavefront: about sqrt(chunks / resident
  // wavefronts), as the pooled lookup chooses its bags per wavefront
  // (EB_BAGS_PER_WAVE fixes it)
  int64_t k = h->bags_per_wave;
  if (k == 0) {
    const int64_t per_slot = ((n + kWave - 1) / kWave) / kResidentWaves;
    k = 1;
    while ((k + 1) * (k + 1) <= per_slot) ++k;
    k = k > kMaxBagsPerWave ? kMaxBagsPerWave : k;
  }
  a.span = (int32_t)(k * kWave);
  a.num_waves = (n + a.span - 1) / a.span;

  hipError_t e = begin_checked(h);
  const unsigned grid = (unsigned)((a.num_waves + kWavesPerBlock - 1) / kWavesPerBlock);
  for (int dt = 0; dt < 3 && e == hipSuccess; ++dt) {
    if (!(h->dtype_mask & (1 << dt))) continue;
    hipLaunchKernelGGL(pick_seq(dt, h->single_log2), dim3(grid), dim3(kBlock), 0, h->stream, a);
    e = hipGetLastError();
  }
  const eb_status st = end_checked(h, e);
  if (cur != h->device) (void)hipSetDevice(cur);
  return st;
}
