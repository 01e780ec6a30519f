// Streaming-read ceiling of the GPU's HBM: a plain kernel that reads a 2 GiB
// buffer once with 16-byte loads (each workgroup one contiguous chunk, UNR
// loads in flight per thread) and writes one word per thread.  It serves as
// the practical upper bound against which the decode-shaped forward (which
// reads K and V once) is judged; it computes nothing of the attention path.
//
// Prints one JSON line per launch shape and a last line with the best.
#include <hip/hip_runtime.h>
#include <stdio.h>
#include <stdlib.h>

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

template <int UNR, bool NT>
__global__ __launch_bounds__(256) void read_chunks(const u32x4* __restrict__ src, unsigned* __restrict__ out,
                                                   size_t per_wg) {
  const u32x4* p = src + (size_t)blockIdx.x * per_wg;
  unsigned acc = 0;
  for (size_t base = 0; base < per_wg; base += 256 * UNR) {
    u32x4 v[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const u32x4* a = p + base + u * 256 + threadIdx.x;
      v[u] = NT ? __builtin_nontemporal_load(a) : *a;
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
  }
  out[(size_t)blockIdx.x * 256 + threadIdx.x] = acc;
}

#define CHECK(x)                                                            \
  do {                                                                      \
    hipError_t e_ = (x);                                                    \
    if (e_ != hipSuccess) {                                                 \
      fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));        \
      return 1;                                                             \
    }                                                                       \
  } while (0)

struct Shape {
  const char* name;
  int wgs, unr;
  void (*kernel)(const u32x4*, unsigned*, size_t);
};

int main() {
  const size_t bytes = (size_t)2 << 30, n16 = bytes / 16;
  const int max_wgs = 16384;
  u32x4* src = nullptr;
  unsigned* out = nullptr;
  CHECK(hipMalloc(&src, bytes));
  CHECK(hipMemset(src, 1, bytes));
  CHECK(hipMalloc(&out, (size_t)max_wgs * 256 * sizeof(unsigned)));
  hipEvent_t a, b;
  CHECK(hipEventCreate(&a));
  CHECK(hipEventCreate(&b));
  const Shape shapes[] = {
      {"wg2048_unr8", 2048, 8, read_chunks<8, false>},   {"wg4096_unr8", 4096, 8, read_chunks<8, false>},
      {"wg8192_unr8", 8192, 8, read_chunks<8, false>},   {"wg16384_unr8", 16384, 8, read_chunks<8, false>},
      {"wg8192_unr16", 8192, 16, read_chunks<16, false>}, {"wg8192_unr8_nt", 8192, 8, read_chunks<8, true>},
      {"wg2048_unr8_nt", 2048, 8, read_chunks<8, true>},
  };
  double best = 0.0;
  const char* best_name = "";
  for (const Shape& s : shapes) {
    // Every shape divides the buffer into equal chunks of whole load rounds.
    const size_t per_wg = n16 / (size_t)s.wgs;
    if (s.wgs > max_wgs || per_wg * (size_t)s.wgs != n16 || per_wg % (size_t)(256 * s.unr) != 0) {
      fprintf(stderr, "shape %s does not tile the buffer\n", s.name);
      return 1;
    }
    const int warm = 3, reps = 20;
    float times[reps];
    for (int r = 0; r < warm + reps; ++r) {
      CHECK(hipEventRecord(a, 0));
      hipLaunchKernelGGL(s.kernel, dim3((unsigned)s.wgs), dim3(256), 0, 0, src, out, per_wg);
      CHECK(hipGetLastError());
      CHECK(hipEventRecord(b, 0));
      CHECK(hipEventSynchronize(b));
      float ms = 0.0f;
      CHECK(hipEventElapsedTime(&ms, a, b));
      if (r >= warm) times[r - warm] = ms;
    }
    // median of the timed launches
    for (int i = 1; i < reps; ++i)
      for (int j = i; j > 0 && times[j - 1] > times[j]; --j) {
        const float t = times[j];
        times[j] = times[j - 1];
        times[j - 1] = t;
      }
    const double med = 0.5 * (times[reps / 2 - 1] + times[reps / 2]);
    const double gbps = (double)bytes / (med * 1e-3) / 1e9;
    printf("{\"shape\": \"%s\", \"bytes\": %zu, \"median_ms\": %.4f, \"GBps\": %.1f, \"frac_of_8TBps\": %.4f}\n",
           s.name, bytes, med, gbps, gbps / 8000.0);
    if (gbps > best) {
      best = gbps;
      best_name = s.name;
    }
  }
  printf("{\"best_shape\": \"%s\", \"GBps\": %.1f, \"frac_of_8TBps\": %.4f}\n", best_name, best, best / 8000.0);
  CHECK(hipFree(src));
  CHECK(hipFree(out));
  return 0;
}
