// Streaming-read reference for the decode kernels' roofline: how fast one
// launch that only reads N MiB (16-byte nontemporal loads, each work-group one
// contiguous chunk, 8 loads in flight per thread) runs on this GPU, for the
// byte counts the decode kernels move.  Times are dispatch-stamped events
// (kernel start to end), averaged over 50 launches that rotate over 2 GB so no
// launch is served from the last-level cache.  Not part of the library.
//
//   stream_probe            prints one line per (MiB, work-groups) pair
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <vector>

#define CHECK(x)                                                                      \
  do {                                                                                \
    hipError_t e_ = (x);                                                              \
    if (e_ != hipSuccess) {                                                           \
      std::fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));             \
      std::exit(1);                                                                   \
    }                                                                                 \
  } while (0)

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

template <int U>
__global__ __launch_bounds__(256) void stream_read(const u32x4* __restrict__ src, size_t chunk_vec, uint32_t* out) {
  const u32x4* p = src + blockIdx.x * chunk_vec;
  uint32_t acc = 0;
  for (size_t i = threadIdx.x; i < chunk_vec; i += 256 * U) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      v[u] = (i + u * 256 < chunk_vec) ? __builtin_nontemporal_load(p + i + u * 256) : u32x4{0, 0, 0, 0};
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
  }
  out[blockIdx.x * 256 + threadIdx.x] = acc;  // keeps the loads
}

int main() {
  const size_t total = size_t{2} << 30;
  const int reps = 50;
  char* buf;
  uint32_t* out;
  CHECK(hipMalloc(&buf, total));
  CHECK(hipMalloc(&out, size_t{4096} * 256 * sizeof(uint32_t)));
  CHECK(hipMemset(buf, 1, total));
  std::vector<hipEvent_t> e0(reps), e1(reps);
  for (int i = 0; i < reps; ++i) {
    CHECK(hipEventCreate(&e0[i]));
    CHECK(hipEventCreate(&e1[i]));
  }
  for (size_t mib : {48, 60, 64, 96, 128, 256, 512}) {
    const size_t bytes = mib << 20;
    const size_t nrot = total / bytes;
    for (int nwg : {256, 512, 1024, 2048, 4096}) {
      const size_t chunk = bytes / nwg;
      if (chunk % 4096 != 0) continue;
      auto launch = [&](int r, hipEvent_t a, hipEvent_t b) {
        const u32x4* src = reinterpret_cast<const u32x4*>(buf + (r % nrot) * bytes);
        hipExtLaunchKernelGGL((stream_read<8>), dim3(nwg), dim3(256), 0, 0, a, b, 0, src, chunk / 16, out);
      };
      for (int i = 0; i < 4; ++i) launch(i, nullptr, nullptr);
      CHECK(hipDeviceSynchronize());
      for (int i = 0; i < reps; ++i) launch(i + 4, e0[i], e1[i]);
      CHECK(hipDeviceSynchronize());
      std::vector<float> ms(reps);
      for (int i = 0; i < reps; ++i) CHECK(hipEventElapsedTime(&ms[i], e0[i], e1[i]));
      double mean = 0;
      for (float t : ms) mean += t;
      mean /= reps;
      std::sort(ms.begin(), ms.end());
      std::printf("stream %4zu MiB nwg %5d  mean %8.2f us  median %8.2f us  min %8.2f us  %6.0f GB/s  %5.1f%% of 8 TB/s\n",
                  mib, nwg, mean * 1e3, ms[reps / 2] * 1e3, ms[0] * 1e3, bytes / (mean * 1e-3) / 1e9,
                  100.0 * bytes / (mean * 1e-3) / 8e12);
      std::fflush(stdout);
    }
  }
  return 0;
}
