// Issue-rate probe for the gfx950 facts the kernels are designed around (no
// attention arithmetic).  Two parts, timed with s_memtime inside the kernel:
//
// 1. Cycles per wave64 instruction for v_exp_f32, v_fma_f32,
//    v_dot2c_f32_bf16 and mixes of exponentials and FMAs, one wave per SIMD
//    on every SIMD, 16 independent chains per lane.
// 2. The issue cost of a burst of four 1 KiB global -> LDS copies
//    (global_load_lds_dwordx4) or four 16-byte register loads, issued by waves
//    0-3 of a 512-thread workgroup while waves 4-7 (the same four SIMDs) stay
//    idle, read LDS, or issue MFMAs.
//
// Prints one JSON line per measurement.
#include <hip/hip_runtime.h>
#include <stdio.h>
#include <stdlib.h>

typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

#define CHECK(x)                                                            \
  do {                                                                      \
    hipError_t e_ = (x);                                                    \
    if (e_ != hipSuccess) {                                                 \
      fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));        \
      exit(1);                                                              \
    }                                                                       \
  } while (0)

// ------------------------------------------------------------ part 1
constexpr int kIter = 2048;
template <int MODE>
__global__ __launch_bounds__(256) void valu_rates(float* out, float seed, long long* cyc) {
  float x[16], y[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    x[i] = seed * (i + 1) + threadIdx.x * 1e-3f;
    y[i] = x[i] * 0.5f;
  }
  const bf2 one = {(__bf16)1.0f, (__bf16)1.0f};
  const long long t0 = __builtin_amdgcn_s_memtime();
  for (int it = 0; it < kIter; ++it) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (MODE == 0) x[i] = __builtin_amdgcn_exp2f(x[i]);
      if (MODE == 1) x[i] = __builtin_fmaf(x[i], 0.999f, 1e-3f);
      if (MODE == 2) {
        x[i] = __builtin_amdgcn_exp2f(x[i]);
        y[i] = __builtin_fmaf(y[i], 0.999f, 1e-3f);
      }
      if (MODE == 3) y[i] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf2, x[i]), one, y[i], false);
      if (MODE == 4) {
        x[i] = __builtin_amdgcn_exp2f(x[i]);
        y[i] = __builtin_fmaf(y[i], 0.999f, 1e-3f);
        y[i] = __builtin_fmaf(y[i], 0.998f, 1e-3f);
        y[i] = __builtin_fmaf(y[i], 0.997f, 1e-3f);
      }
    }
    __asm__ volatile("" ::: "memory");
  }
  const long long t1 = __builtin_amdgcn_s_memtime();
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) s += x[i] + y[i];
  const int g = blockIdx.x * blockDim.x + threadIdx.x;
  out[g] = s;
  if ((threadIdx.x & 63) == 0) cyc[g >> 6] = t1 - t0;
}

template <int MODE>
void run_valu(const char* name, double per, float* out, long long* cyc, long long* h) {
  const int blocks = 256;  // 1024 waves: one per SIMD
  for (int r = 0; r < 2; ++r) hipLaunchKernelGGL(valu_rates<MODE>, dim3(blocks), dim3(256), 0, 0, out, 0.25f, cyc);
  CHECK(hipGetLastError());
  CHECK(hipDeviceSynchronize());
  CHECK(hipMemcpy(h, cyc, blocks * 4 * sizeof(long long), hipMemcpyDeviceToHost));
  double sum = 0;
  for (int i = 0; i < blocks * 4; ++i) sum += (double)h[i];
  printf("{\"part\": \"valu\", \"what\": \"%s\", \"memtime_ticks\": %.2f}\n", name, sum / (blocks * 4) / (16.0 * kIter) * per);
}

// ------------------------------------------------------------ part 2
constexpr int kReps = 256;
constexpr size_t kRegion = 262144;  // source bytes per workgroup
template <int OTHER, bool VGPR>
__global__ __launch_bounds__(512) void copy_issue(const unsigned char* __restrict__ src, float* out, long long* cyc) {
  __shared__ __align__(16) unsigned char lds[64 * 1024];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const unsigned char* base = src + (size_t)blockIdx.x * kRegion;
  long long tsum = 0;
  float acc = 0.0f;
  if (wave < 4) {
    u32x4 r[4];
    for (int it = 0; it < kReps; ++it) {
      // a 4 KiB burst at one of 62 positions: offset + 4 KiB <= 62 * 4 KiB < kRegion
      const unsigned char* g = base + ((it * 4 + wave) % 62) * 4096;
      __builtin_amdgcn_sched_barrier(0);
      const long long t0 = __builtin_amdgcn_s_memtime();
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        if (VGPR) {
          r[c] = *reinterpret_cast<const u32x4*>(g + c * 1024 + lane * 16);
        } else {
          // LDS destination: wave * 16 KiB + c KiB + 16 * lane < 64 KiB
          const unsigned dst = __builtin_amdgcn_readfirstlane((unsigned)(size_t)lds + wave * 16384 + c * 1024);
          const void* a = g + c * 1024 + lane * 16;
          asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                       :
                       : "v"(a), "s"(dst)
                       : "memory", "m0");
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      const long long t1 = __builtin_amdgcn_s_memtime();
      __builtin_amdgcn_sched_barrier(0);
      tsum += t1 - t0;
      for (int i = 0; i < 64; ++i) acc = __builtin_fmaf(acc, 0.999f, 1e-3f);
      __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
      if (VGPR) {
#pragma unroll
        for (int c = 0; c < 4; ++c) acc += __uint_as_float(r[c][0] & 0x3f800000u);
      }
    }
  } else if (OTHER == 1) {  // LDS reads of the upper 32 KiB
    for (int it = 0; it < kReps * 8; ++it) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(lds + 32768 + ((it * 64 + lane) % 2048) * 16);
      acc += __uint_as_float(v[0] & 0x3f800000u);
    }
  } else if (OTHER == 2) {  // back-to-back MFMAs
    f32x16 c = {};
    bf16x8 a, b;
    for (int e = 0; e < 8; ++e) {
      a[e] = (__bf16)(lane * 0.01f);
      b[e] = (__bf16)(e * 0.1f);
    }
    for (int it = 0; it < kReps * 8; ++it) c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
    acc = c[0];
  }
  __syncthreads();
  out[blockIdx.x * 512 + threadIdx.x] = acc + lds[threadIdx.x];
  if (lane == 0) cyc[blockIdx.x * 8 + wave] = tsum;
}

template <int OTHER, bool VGPR>
void run_copy(const char* name, const unsigned char* src, float* out, long long* cyc, long long* h) {
  for (int r = 0; r < 3; ++r)
    hipLaunchKernelGGL((copy_issue<OTHER, VGPR>), dim3(256), dim3(512), 0, 0, src, out, cyc);
  CHECK(hipGetLastError());
  CHECK(hipDeviceSynchronize());
  CHECK(hipMemcpy(h, cyc, 256 * 8 * sizeof(long long), hipMemcpyDeviceToHost));
  double s = 0;
  for (int b = 0; b < 256; ++b)
    for (int w = 0; w < 4; ++w) s += (double)h[b * 8 + w];
  printf("{\"part\": \"issue\", \"what\": \"%s\", \"memtime_ticks_per_burst_of_4\": %.1f}\n", name, s / 1024 / kReps);
}

int main() {
  float* out = nullptr;
  long long* cyc = nullptr;
  unsigned char* src = nullptr;
  long long* h = (long long*)malloc(256 * 8 * sizeof(long long));
  CHECK(hipMalloc(&out, 256 * 512 * sizeof(float)));
  CHECK(hipMalloc(&cyc, 256 * 8 * sizeof(long long)));
  CHECK(hipMalloc(&src, 256 * kRegion));
  CHECK(hipMemset(src, 1, 256 * kRegion));
  run_valu<0>("v_exp_f32 per instruction", 1.0, out, cyc, h);
  run_valu<1>("v_fma_f32 per instruction", 1.0, out, cyc, h);
  run_valu<2>("v_exp_f32 + v_fma_f32 (independent chains) per pair", 1.0, out, cyc, h);
  run_valu<3>("v_dot2c_f32_bf16 per instruction", 1.0, out, cyc, h);
  run_valu<4>("v_exp_f32 + 3 v_fma_f32 per group", 1.0, out, cyc, h);
  run_copy<0, false>("4 global->LDS copies, other waves idle", src, out, cyc, h);
  run_copy<1, false>("4 global->LDS copies, other waves reading LDS", src, out, cyc, h);
  run_copy<2, false>("4 global->LDS copies, other waves issuing MFMAs", src, out, cyc, h);
  run_copy<0, true>("4 register loads, other waves idle", src, out, cyc, h);
  run_copy<2, true>("4 register loads, other waves issuing MFMAs", src, out, cyc, h);
  CHECK(hipFree(out));
  CHECK(hipFree(cyc));
  CHECK(hipFree(src));
  free(h);
  return 0;
}
