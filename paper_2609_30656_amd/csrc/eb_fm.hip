// libeb — the factorization-machine cross term over the pooled embeddings.
//
// The paper's DLRM is DeepFM-based: its inter_arch.fm submodule takes the
// pooled embeddings that sparse_arch produces and computes the FM cross term,
// a few small element-wise passes and reductions that the paper finds
// bandwidth-bound (Sec. IV-A.2, inter_arch zoom-in).  Its value per example b
// is the FM second-order term over fields (Rendle 2010, cited in the
// Introduction) with field f's pooled embedding e_f as its factor vector:
//
//   y_b = sum_{f < f'} <e_f, e_f'> = 1/2 sum_d [ (sum_f e_{f,d})^2 - sum_f e_{f,d}^2 ]
//
// One pass over the pooled output [B, T*D] (each byte read once, y written
// once), one wavefront per example.  The example's T fields are rows of D
// fp32 values, gathered like table rows: 16-byte lane slices, LPR lanes per
// field, RPL = 64 / LPR fields per wave-wide load, several loads in flight.
// Each lane keeps sum_f e and sum_f e^2 for its slice; the forward's
// reduce-scatter combines the row groups in a fixed order, and a butterfly
// sums (sum e)^2 - sum e^2 over the columns, so y is deterministic.
//
// Why not inside the lookup kernel: the lookup walks its bags table by table,
// so at any time only a few tables' hot rows compete for L2 and the Infinity
// Cache.  Forming y in registers needs all T tables of an example at once;
// walked that way (example by example) the lookup ran 1.3-1.5x slower on
// MI355X, far more than this pass costs (at most 10% of the lookup's time on
// the measured workloads).

#include "eb_device.h"

namespace eb {
namespace {

struct FmArgs {
  const float *pooled;  // [batch, ld]: field f of example b at pooled[b*ld + f*dim]
  float *fm;            // [batch]
  const float *zero;    // all-zero row
  int64_t ld;
  int32_t batch;
  int32_t fields;
  int32_t dim;
  int32_t passes;       // 256-value column windows per field
};

constexpr int kFmWindow = kPassBytes / 4;  // fp32 values per column window

// Fields [(s0 + u) * RPL + grp] for u < N of this lane's column slice, added
// into the running sums s and s2 (straight-line: missing fields read the zero
// row, so all N loads are in flight together).
template <int LPR, int N>
__device__ __forceinline__ void fm_steps(const FmArgs &a, const float *row, int col, bool colok, int s0,
                                         float (&s)[4], float (&s2)[4]) {
  constexpr int RPL = kWave / LPR;
  const int grp = (threadIdx.x & (kWave - 1)) / LPR;
  f32x4 v[N];
#pragma unroll
  for (int u = 0; u < N; ++u) {
    const int f = (s0 + u) * RPL + grp;
    const float *p = (f < a.fields && colok) ? row + (int64_t)f * a.dim + col : a.zero;
    v[u] = *(const EB_GLOBAL f32x4 *)p;  // a global-memory load, not a flat one
  }
#pragma unroll
  for (int u = 0; u < N; ++u) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      s[i] += v[u][i];
      s2[i] = fmaf(v[u][i], v[u][i], s2[i]);
    }
  }
}

// U: steps per batch.  An example of at most 4 steps takes the same batch of
// 4 either way; compiled for U = 4 the kernel needs 52 VGPRs rather than 88
// (8 waves per SIMD rather than 5), which took 8 fields of 128 values at
// batch 16 384 from 11.4 to 11.0 us on MI355X.
template <int LOG2, int U>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(U == 4 ? 8 : 1, 8))) void eb_fm_kernel(
    FmArgs a) {
  constexpr int LPR = 1 << LOG2;
  constexpr int RPL = kWave / LPR;
  using R = Reduce<kF32, LPR>;
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t b = (int64_t)blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  if (b >= a.batch) return;
  const float *row = a.pooled + b * a.ld;
  const int steps = (a.fields + RPL - 1) / RPL;

  float y = 0.0f;
  for (int p = 0; p < a.passes; ++p) {
    const int col = p * kFmWindow + (lane % LPR) * 4;
    const bool colok = col < a.dim;
    float s[4] = {0.0f, 0.0f, 0.0f, 0.0f}, s2[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    int st = 0;
    for (; steps - st > U / 2; st += U) fm_steps<LPR, U>(a, row, col, colok, st, s, s2);
    const int rem = steps - st;  // 0 .. U/2
    if (rem > 2) fm_steps<LPR, 4>(a, row, col, colok, st, s, s2);
    else if (rem == 2) fm_steps<LPR, 2>(a, row, col, colok, st, s, s2);
    else if (rem == 1) fm_steps<LPR, 1>(a, row, col, colok, st, s, s2);
    R::run(s);
    R::run(s2);
    if (R::stores(lane) && colok) {
      // no fma: (sum e)^2 is rounded on its own, as each e^2 in s2 was, so
      // with a single field the two cancel exactly and the term is 0
#pragma clang fp contract(off)
#pragma unroll
      for (int i = 0; i < R::KEEP; ++i) y += s[i] * s[i] - s2[i];
    }
  }
#pragma unroll
  for (int o = kWave / 2; o >= 1; o >>= 1) y += __shfl_xor(y, o);
  if (lane == 0) a.fm[b] = 0.5f * y;
}

typedef void (*FmKernelFn)(FmArgs);

template <int U>
FmKernelFn pick_fm_u(int log2) {
  switch (log2) {
    case 0: return eb_fm_kernel<0, U>;
    case 1: return eb_fm_kernel<1, U>;
    case 2: return eb_fm_kernel<2, U>;
    case 3: return eb_fm_kernel<3, U>;
    case 4: return eb_fm_kernel<4, U>;
    case 5: return eb_fm_kernel<5, U>;
    default: return eb_fm_kernel<6, U>;
  }
}

FmKernelFn pick_fm(int log2, int steps) { return steps > 4 ? pick_fm_u<8>(log2) : pick_fm_u<4>(log2); }

// Checks shared by both entry points: fm_out is fp32 [batch] and every table
// has the same width.
eb_status check_fm_args(const eb_tables *h, const eb_tensor &fm_out, int64_t batch) {
  if (fm_out.elem_type != EB_T_F32) return EB_ERR_DTYPE;
  if (!fm_out.data) return EB_ERR_INVALID_ARG;
  if (h->uniform_dim == 0 || fm_out.numel != batch) return EB_ERR_SHAPE;
  if (reinterpret_cast<uintptr_t>(fm_out.data) % 4 != 0) return EB_ERR_UNSUPPORTED;
  return EB_OK;
}

hipError_t launch_fm(const eb_tables *h, const float *pooled, int64_t batch, float *fm) {
  FmArgs a;
  a.pooled = pooled;
  a.fm = fm;
  a.zero = reinterpret_cast<const float *>(h->d_zero);
  a.ld = h->sum_dim;
  a.batch = (int32_t)batch;
  a.fields = h->num_tables;
  a.dim = h->uniform_dim;
  a.passes = (a.dim + kFmWindow - 1) / kFmWindow;
  const int log2 = log2_lanes_per_row(4 * (a.dim < kFmWindow ? a.dim : kFmWindow));
  const int steps = (a.fields + (kWave >> log2) - 1) / (kWave >> log2);  // wave-wide loads per example
  const unsigned grid = (unsigned)((batch + kWavesPerBlock - 1) / kWavesPerBlock);
  hipLaunchKernelGGL(pick_fm(log2, steps), dim3(grid), dim3(kBlock), 0, h->stream, a);
  return hipGetLastError();
}

}  // namespace
}  // namespace eb

using namespace eb;

extern "C" {

eb_status eb_fm_cross(const eb_tables *h, eb_tensor pooled, eb_tensor fm_out) {
  if (!h) return EB_ERR_INVALID_ARG;
  if (pooled.elem_type != EB_T_F32) return EB_ERR_DTYPE;
  if (!pooled.data) return EB_ERR_INVALID_ARG;
  if (pooled.numel < h->sum_dim || pooled.numel % h->sum_dim != 0) return EB_ERR_SHAPE;
  const int64_t batch = pooled.numel / h->sum_dim;
  if (batch > INT32_MAX) return EB_ERR_SHAPE;
  const eb_status chk = check_fm_args(h, fm_out, batch);
  if (chk != EB_OK) return chk;
  if (reinterpret_cast<uintptr_t>(pooled.data) % 16 != 0) return EB_ERR_UNSUPPORTED;

  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return EB_ERR_HIP;
  if (cur != h->device && hipSetDevice(h->device) != hipSuccess) return EB_ERR_HIP;
  const hipError_t e = launch_fm(h, static_cast<const float *>(pooled.data), batch,
                                 static_cast<float *>(const_cast<void *>(fm_out.data)));
  if (cur != h->device) (void)hipSetDevice(cur);
  return e == hipSuccess ? EB_OK : EB_ERR_HIP;
}

eb_status eb_forward_fm(const eb_tables *h, eb_tensor indices, eb_tensor offsets, eb_tensor per_sample_weights,
                        eb_pooling pooling, eb_tensor out, eb_tensor fm_out) {
  FwdShape sh;
  eb_status chk = check_forward_args(h, indices, offsets, per_sample_weights, pooling, out, &sh);
  if (chk != EB_OK) return chk;
  chk = check_fm_args(h, fm_out, sh.batch);
  if (chk != EB_OK) return chk;

  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return EB_ERR_HIP;
  if (cur != h->device && hipSetDevice(h->device) != hipSuccess) return EB_ERR_HIP;
  hipError_t e = begin_checked(h);
  if (e == hipSuccess) e = launch_forward(h, indices, offsets, per_sample_weights, pooling, out, sh);
  if (e == hipSuccess)
    e = launch_fm(h, static_cast<const float *>(out.data), sh.batch,
                  static_cast<float *>(const_cast<void *>(fm_out.data)));
  const eb_status st = end_checked(h, e);
  if (cur != h->device) (void)hipSetDevice(cur);
  return st;
}

}  // extern "C"
