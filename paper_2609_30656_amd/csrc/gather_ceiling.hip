// gather_ceiling — the random-row gather rate this GPU sustains, the practical
// ceiling for a lookup whose rows miss every cache.
//
//   paper_2609_30656_amd/gather_ceiling            (built with libeb.so)
//
// Each wavefront reads rows of ROW bytes at random row indices (drawn on the
// host, every one below the row count) from a 16 GiB buffer, 16 bytes per
// lane, U wave-wide loads in flight per lane, and writes one checksum word
// per wavefront.  The bytes moved per launch are the rows' bytes (the 4-byte
// indices add 4 / ROW).  One line per (ROW, U): the launch time averaged
// over 10 launches after 3 warm-up launches, and the row bytes per second.
// The 8 TB/s HBM peak is a streaming rate; this is what random rows reach.

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <random>
#include <vector>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kWaves = 4;  // wavefronts per workgroup

template <int ROW, int U>
__global__ __launch_bounds__(kWave * kWaves) void gather(const unsigned char *__restrict__ buf,
                                                         const uint32_t *__restrict__ idx, int64_t slots,
                                                         uint32_t *out, int per_wave) {
  constexpr int LPR = ROW / 16;      // lanes per row
  constexpr int RPL = kWave / LPR;   // rows per wave-wide load
  const int lane = threadIdx.x % kWave;
  const int64_t wave = (int64_t)blockIdx.x * kWaves + threadIdx.x / kWave;
  const int64_t first = wave * per_wave;
  uint32_t acc = 0;
  for (int s = 0; s < per_wave; s += U * RPL) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      int64_t slot = first + s + u * RPL + lane / LPR;
      if (slot >= slots) slot = slots - 1;
      v[u] = *(const u32x4 *)(buf + (uint64_t)idx[slot] * ROW + (lane % LPR) * 16);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  if (lane == 0) out[wave] = acc;
}

bool ok(hipError_t e, const char *what) {
  if (e != hipSuccess) fprintf(stderr, "gather_ceiling: %s: %s\n", what, hipGetErrorString(e));
  return e == hipSuccess;
}

template <int ROW, int U>
bool run(const unsigned char *buf, size_t bytes, uint32_t *didx, uint32_t *dout, int64_t slots) {
  const uint64_t rows = bytes / ROW;
  std::vector<uint32_t> h(slots);
  std::mt19937_64 g(ROW * 131 + U);
  for (auto &x : h) x = (uint32_t)(g() % rows);
  if (!ok(hipMemcpy(didx, h.data(), slots * 4, hipMemcpyHostToDevice), "copy indices")) return false;
  const int per_wave = kWave / (ROW / 16) * U * 4;  // four batches of U loads per wavefront
  const int64_t waves = slots / per_wave;           // slots is a multiple of per_wave
  const unsigned grid = (unsigned)(waves / kWaves);
  hipEvent_t a, b;
  if (!ok(hipEventCreate(&a), "event") || !ok(hipEventCreate(&b), "event")) return false;
  for (int rep = 0; rep < 3; ++rep)
    hipLaunchKernelGGL((gather<ROW, U>), dim3(grid), dim3(kWave * kWaves), 0, 0, buf, didx, slots, dout, per_wave);
  constexpr int kReps = 10;
  (void)hipEventRecord(a);
  for (int rep = 0; rep < kReps; ++rep)
    hipLaunchKernelGGL((gather<ROW, U>), dim3(grid), dim3(kWave * kWaves), 0, 0, buf, didx, slots, dout, per_wave);
  (void)hipEventRecord(b);
  if (!ok(hipEventSynchronize(b), "launch")) return false;
  float ms = 0.0f;
  (void)hipEventElapsedTime(&ms, a, b);
  const double moved = (double)grid * kWaves * per_wave * ROW;
  const double s = ms * 1e-3 / kReps;
  printf("row_bytes=%d loads_in_flight=%d launch_us=%.1f row_GBps=%.0f\n", ROW, U, s * 1e6, moved / s / 1e9);
  fflush(stdout);
  (void)hipEventDestroy(a);
  (void)hipEventDestroy(b);
  return true;
}

}  // namespace

int main() {
  const size_t bytes = (size_t)16 << 30;
  const int64_t slots = (int64_t)4 << 20;  // rows per launch (a multiple of every per_wave)
  unsigned char *buf = nullptr;
  uint32_t *didx = nullptr, *dout = nullptr;
  if (!ok(hipMalloc(&buf, bytes), "alloc") || !ok(hipMalloc(&didx, slots * 4), "alloc") ||
      !ok(hipMalloc(&dout, slots * 4), "alloc"))
    return 2;
  if (!ok(hipMemset(buf, 1, bytes), "fill")) return 2;
  bool good = run<128, 8>(buf, bytes, didx, dout, slots) && run<256, 4>(buf, bytes, didx, dout, slots) &&
              run<256, 8>(buf, bytes, didx, dout, slots) && run<256, 16>(buf, bytes, didx, dout, slots) &&
              run<512, 8>(buf, bytes, didx, dout, slots) && run<1024, 8>(buf, bytes, didx, dout, slots);
  (void)hipFree(buf);
  (void)hipFree(didx);
  (void)hipFree(dout);
  return good ? 0 : 1;
}
