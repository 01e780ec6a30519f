// Streaming-read ceiling of the GPU's HBM: plain kernels that read a 2 GiB
// buffer once with 16-byte loads (each workgroup one contiguous chunk, UNR
// loads in flight per thread, or asynchronous copies into an LDS ring) and
// write one word per thread.  It serves as
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

// The same read through asynchronous global -> LDS copies
// (global_load_lds_dwordx4, the path the decode kernel uses), one wave per
// workgroup: each 1 KiB unit lands in a RING-slot LDS ring, and the wave
// waits for the older half of the ring before reusing it.  NT selects the
// non-temporal cache policy.
template <int RING, bool NT>
__global__ __launch_bounds__(64) void read_to_lds(const u32x4* __restrict__ src, unsigned* __restrict__ out,
                                                  size_t per_wg) {
  __shared__ __align__(16) unsigned char ring[RING * 1024];
  const int lane = threadIdx.x;
  const u32x4* p = src + (size_t)blockIdx.x * per_wg;
  const size_t units = per_wg / 64;
  const unsigned base = (unsigned)(size_t)ring;
  for (size_t u = 0; u < units; ++u) {
    const void* a = p + u * 64 + lane;
    const unsigned dst = __builtin_amdgcn_readfirstlane(base + (unsigned)(u % RING) * 1024u);
    if (NT)
      asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt"
                   :
                   : "v"(a), "s"(dst)
                   : "memory", "m0");
    else
      asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                   :
                   : "v"(a), "s"(dst)
                   : "memory", "m0");
    // vmcnt(RING / 2) after every half ring: the slots about to be reused are free.
    // (vmcnt bits 3:0 and 15:14; expcnt and lgkmcnt left unconstrained)
    if (u % (RING / 2) == RING / 2 - 1)
      __builtin_amdgcn_s_waitcnt(0x0F70 | ((RING / 2) & 15) | (((RING / 2) >> 4) << 14));
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);
  __syncthreads();
  out[(size_t)blockIdx.x * 64 + lane] = reinterpret_cast<const unsigned*>(ring)[lane];
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
  int wgs, unr, threads;  // unr: 16-byte loads per thread and round (ring slots for the LDS path)
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
      {"wg2048_unr8", 2048, 8, 256, read_chunks<8, false>},
      {"wg4096_unr8", 4096, 8, 256, read_chunks<8, false>},
      {"wg8192_unr8", 8192, 8, 256, read_chunks<8, false>},
      {"wg16384_unr8", 16384, 8, 256, read_chunks<8, false>},
      {"wg8192_unr16", 8192, 16, 256, read_chunks<16, false>},
      {"wg8192_unr8_nt", 8192, 8, 256, read_chunks<8, true>},
      {"wg2048_unr8_nt", 2048, 8, 256, read_chunks<8, true>},
      {"lds_wg2048_ring16", 2048, 16, 64, read_to_lds<16, false>},
      {"lds_wg2048_ring16_nt", 2048, 16, 64, read_to_lds<16, true>},
      {"lds_wg4096_ring32_nt", 4096, 32, 64, read_to_lds<32, true>},
  };
  double best = 0.0;
  const char* best_name = "";
  for (const Shape& s : shapes) {
    // Every shape divides the buffer into equal chunks of whole load rounds.
    const size_t per_wg = n16 / (size_t)s.wgs;
    if (s.wgs > max_wgs || per_wg * (size_t)s.wgs != n16 || per_wg % (size_t)(s.threads * s.unr) != 0) {
      fprintf(stderr, "shape %s does not tile the buffer\n", s.name);
      return 1;
    }
    const int warm = 3, reps = 20;
    float times[reps];
    for (int r = 0; r < warm + reps; ++r) {
      CHECK(hipEventRecord(a, 0));
      hipLaunchKernelGGL(s.kernel, dim3((unsigned)s.wgs), dim3((unsigned)s.threads), 0, 0, src, out, per_wg);
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
