// Device primitives for the gfx950 (CDNA4) attention kernels: MFMA fragment
// types and wrappers, lane bookkeeping for the 32x32 MFMA tiles, LDS reads
// (plain and transposing), wave-half exchanges and numeric helpers.
//
// MFMA tile conventions used by every kernel (v_mfma_f32_32x32x{16,2}):
//   lane l = 32*h + c with h = l / 32 (lane half) and c = l % 32;
//   A fragment: lane holds A[row c][k = 8h + s], s = 0..7;
//   B fragment: lane holds B[k = 8h + s][col c], s = 0..7;
//   C tile    : lane holds C[row 8*(r/4) + 4h + r%4][col c], r = 0..15.
// A "fragment" is always 8 consecutive k values, so a 16-wide k chunk is one
// 32x32x16 MFMA for 16-bit types and eight 32x32x2 MFMAs for float32 (MFMA s
// consumes element s of both fragments, i.e. the k pair {s, 8 + s}).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mea {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <typename T> struct FragT;
template <> struct FragT<__bf16> { typedef bf16x8 type; typedef bf16x4 half; };
template <> struct FragT<_Float16> { typedef f16x8 type; typedef f16x4 half; };
template <> struct FragT<float> { typedef f32x8 type; typedef f32x4 half; };
template <typename T> using Frag = typename FragT<T>::type;

// C += A * B over a 16-wide k chunk.
__device__ __forceinline__ f32x16 mma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mma(const f16x8& a, const f16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mma(const f32x8& a, const f32x8& b, f32x16 c) {
#pragma unroll
  for (int s = 0; s < 8; ++s) c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[s], b[s], c, 0, 0, 0);
  return c;
}

// Row of the 32x32 C tile held in register r by a lane of half h.
__device__ __forceinline__ constexpr int c_row(int r, int h) { return 8 * (r / 4) + 4 * h + (r % 4); }

// Row permutation applied when an operand's rows are read into an A (or B)
// fragment: with A row i taken from source row perm32(i), register r of lane
// half h in the C tile holds source row 16*(r/8) + 8h + (r%8).  Registers
// 8m..8m+7 of a lane then cover 8 consecutive source rows (16m + 8h + s), which
// is exactly the k layout of a fragment: a C tile can feed the next MFMA as a
// B (or A) operand with no data movement between lanes.
__device__ __forceinline__ constexpr int perm32(int i) {
  return 16 * ((i >> 3) >> 1) + 8 * ((i >> 2) & 1) + 4 * ((i >> 3) & 1) + (i & 3);
}
__device__ __forceinline__ constexpr int permuted_row(int r, int h) { return 16 * (r / 8) + 8 * h + (r % 8); }

// Eight consecutive elements from LDS (16 B for 16-bit types, 32 B for float).
template <typename T>
__device__ __forceinline__ Frag<T> lds_frag(const T* p) {
  return *reinterpret_cast<const Frag<T>*>(p);
}

// Transposing LDS read (ds_read_b64_tr_b16).  Within each group of 16 lanes,
// lane i supplies an 8-byte address e_i and receives element (i % 4) of the
// four chunks e_{4r + i/4}, r = 0..3.  With lane i pointing at
// row (base_row + i/4), column (base_col + 4*(i%4)) of a row-major tile, lane
// i receives column base_col + i of rows base_row .. base_row + 3.
typedef short v4s_t __attribute__((__vector_size__(4 * sizeof(short))));
__device__ __forceinline__ v4s_t lds_read_tr16(const void* p) {
  typedef __attribute__((address_space(3))) v4s_t lds_v4s;
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_v4s*)((__attribute__((address_space(3))) char*)((__attribute__((address_space(3))) void*)p)));
}

// Column fragment of a row-major 16-bit tile: lane (h, c) gets column col0 + c
// of rows row0 + 8h + s, s = 0..7 (rs = row stride in elements).  Lanes are
// grouped by 16: group g covers columns col0 + 16*(g%2) + 0..15, lane half g/2.
template <typename T>
__device__ __forceinline__ Frag<T> lds_col_frag(const T* tile, int rs, int row0, int col0, int lane) {
  static_assert(sizeof(T) == 2, "transposing read is for 16-bit elements");
  const int g = lane >> 4, i = lane & 15;
  const int row = row0 + 8 * (g >> 1) + (i >> 2);
  const int col = col0 + 16 * (g & 1) + 4 * (i & 3);
  const v4s_t lo = lds_read_tr16(tile + row * rs + col);
  const v4s_t hi = lds_read_tr16(tile + (row + 4) * rs + col);
  typedef short v8s_t __attribute__((ext_vector_type(8)));
  v8s_t r;
  r[0] = lo[0]; r[1] = lo[1]; r[2] = lo[2]; r[3] = lo[3];
  r[4] = hi[0]; r[5] = hi[1]; r[6] = hi[2]; r[7] = hi[3];
  return __builtin_bit_cast(Frag<T>, r);
}

// Float32 column fragment: eight scalar reads.
__device__ __forceinline__ f32x8 lds_col_frag_f32(const float* tile, int rs, int row0, int col0, int lane) {
  const int h = lane >> 5, c = lane & 31;
  f32x8 r;
#pragma unroll
  for (int s = 0; s < 8; ++s) r[s] = tile[(row0 + 8 * h + s) * rs + col0 + c];
  return r;
}

// Value of x in the lane of the other half (l ^ 32), via v_permlane32_swap:
// for l < 32 the pair is (x[l], x[l+32]); for l >= 32 it is (x[l-32], x[l]).
__device__ __forceinline__ float xhalf_max(float x) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
}
__device__ __forceinline__ float xhalf_sum(float x) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Wait until every outstanding global load of this wave has completed
// (s_waitcnt vmcnt(0), other counters unconstrained).  Issued once after the
// loads of a kernel's register-resident operands, so that the main loop does
// not re-wait for them -- the counter is in order, and a wait for an early
// load inside the loop would also drain the prefetch of the next tile.
__device__ __forceinline__ void wait_global_loads() { __builtin_amdgcn_s_waitcnt(0x0F70); }
// Wait until at most N vector-memory operations of this wave are in flight
// (they complete in issue order).
template <int N>
__device__ __forceinline__ void wait_global_loads_upto() {
  static_assert(N >= 0 && N < 64, "vmcnt immediate");
  // vmcnt bits 3:0 and 15:14, expcnt 6:4 and lgkmcnt 11:8 left unconstrained.
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}
// The same with a wave-uniform runtime count n <= NMAX.
template <int NMAX>
__device__ __forceinline__ void wait_global_loads_rt(int n) {
  if constexpr (NMAX <= 0) {
    wait_global_loads();
  } else {
    if (n >= NMAX) wait_global_loads_upto<NMAX>();
    else wait_global_loads_rt<NMAX - 1>(n);
  }
}
// Wait until every LDS read of this wave has returned (lgkmcnt(0), vmcnt and
// expcnt unconstrained): the LDS space they read may then be overwritten.
__device__ __forceinline__ void wait_lds_reads() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// Materialise v in registers at this point: an empty statement that takes v
// as input, so that the computation of v cannot be sunk past what follows
// (for example past a barrier into the next phase of a phase-split kernel).
template <typename V>
__device__ __forceinline__ void keep_here(const V& v) {
  asm volatile("" ::"v"(v));
}

// Wave issue priority for the phase-split kernels: the wave in its MFMA phase
// is raised above the wave in its softmax phase on the same SIMD, so that the
// arbiter, which otherwise favours the older wave, issues each MFMA as soon as
// the matrix pipe can take it and the softmax wave fills the remaining slots.
#ifndef MEA_PP_PRIO
#define MEA_PP_PRIO 1
#endif
__device__ __forceinline__ void mfma_phase_priority() {
  if (MEA_PP_PRIO) __builtin_amdgcn_s_setprio(MEA_PP_PRIO);
}
__device__ __forceinline__ void valu_phase_priority() {
  if (MEA_PP_PRIO) __builtin_amdgcn_s_setprio(0);
}

// LDS byte address of a pointer into shared memory (the low 32 bits of its
// generic address).
__device__ __forceinline__ unsigned lds_addr(const void* p) {
  return static_cast<unsigned>(reinterpret_cast<uintptr_t>(p));
}

// Asynchronous copy global -> LDS of 16 bytes per lane (global_load_lds_dwordx4):
// lane l's bytes land at lds_base + 16 l, lds_base being wave-uniform.  It is
// issued from inline assembly so that the compiler adds no waits of its own
// for it: the caller waits (wait_global_loads) and synchronises before the
// data is read.  M0 carries the LDS address and needs one wait state before
// the copy that reads it.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// NT selects the non-temporal cache policy, for data read exactly once (the
// decode kernel's K and V): a streaming read through it measured 7.0 TB/s
// against 6.0 TB/s with the default policy on the same buffer.
template <bool NT = false>
__device__ __forceinline__ void copy_to_lds16(const void* src, unsigned lds_base) {
  if constexpr (NT)
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt"
                 :
                 : "v"(src), "s"(lds_base)
                 : "memory", "m0");
  else
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :
                 : "v"(src), "s"(lds_base)
                 : "memory", "m0");
}
// The same copy with a wave-uniform base address in SGPRs and a per-lane
// 32-bit byte offset (lane l reads base + voff_l): a tile's copies then cost
// no vector instructions beyond the offsets computed once.
template <bool NT = false>
__device__ __forceinline__ void copy_to_lds16_sb(const void* base, unsigned voff, unsigned lds_base) {
  // readfirstlane returns int: widen each half as unsigned (a sign-extended
  // low half would corrupt the high half).
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  const unsigned hi = static_cast<unsigned>(__builtin_amdgcn_readfirstlane(static_cast<unsigned>(b >> 32)));
  const unsigned lo = static_cast<unsigned>(__builtin_amdgcn_readfirstlane(static_cast<unsigned>(b)));
  const uint64_t sb = (static_cast<uint64_t>(hi) << 32) | static_cast<uint64_t>(lo);
  if constexpr (NT)
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 nt"
                 :
                 : "v"(voff), "s"(sb), "s"(lds_base)
                 : "memory", "m0");
  else
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(voff), "s"(sb), "s"(lds_base)
                 : "memory", "m0");
}
#pragma clang diagnostic pop

// Convert eight float32 values to a fragment of T (round to nearest even).
template <typename T>
__device__ __forceinline__ Frag<T> to_frag(const float* x) {
  Frag<T> r;
#pragma unroll
  for (int s = 0; s < 8; ++s) r[s] = (T)x[s];
  return r;
}

// Two float32 values rounded to T (nearest even) and packed low, high.
template <typename T>
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  static_assert(sizeof(T) == 2, "16-bit types only");
  typedef T t2 __attribute__((ext_vector_type(2)));
  const t2 v = {(T)a, (T)b};
  return __builtin_bit_cast(uint32_t, v);
}

// acc + the sum of n weights, added as a balanced tree so that the
// dependency chain is log2(n) + 1 additions long.  The denominator adds the
// float32 weights before they are rounded for the PV MFMA: the difference is
// one rounding per weight, of random sign, far below the 16-bit rounding of
// the products themselves.  (Packed dot products of the rounded fragment with
// 1 would add exactly the rounded weights, but on gfx950 they cost several
// times a VALU add while MFMAs are in flight.)
template <int N>
__device__ __forceinline__ float tree_sum(const float* x, float acc) {
  static_assert(N == 4 || N == 8, "4 or 8 terms");
  if constexpr (N == 4) {
    return acc + ((x[0] + x[1]) + (x[2] + x[3]));
  } else {
    return acc + (((x[0] + x[1]) + (x[2] + x[3])) + ((x[4] + x[5]) + (x[6] + x[7])));
  }
}

// Four float32 results stored as TO at og.  For a 16-bit TO with a residual
// buffer (lo != null) their rounding residuals x - (float)(TO)x, themselves
// rounded to TO, go to lo: the difference of a float32 value and its 16-bit
// rounding is exact in float32, so the pair carries about twice the 16-bit
// precision.
template <typename TO>
__device__ __forceinline__ void store_out4(TO* og, TO* lo, const float (&x)[4]) {
  typedef typename FragT<TO>::half H4;
  H4 v4;
#pragma unroll
  for (int e = 0; e < 4; ++e) v4[e] = (TO)x[e];
  *reinterpret_cast<H4*>(og) = v4;
  if constexpr (sizeof(TO) == 2) {
    if (lo) {
      H4 r4;
#pragma unroll
      for (int e = 0; e < 4; ++e) r4[e] = (TO)(x[e] - (float)v4[e]);
      *reinterpret_cast<H4*>(lo) = r4;
    }
  }
}

// 16-byte global load / store helpers.
__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }

// 16/sizeof(T) consecutive elements read from an array of TO and returned in
// T format (TO is T, or float for a 16-bit T: 32 bytes read and rounded).
template <typename T, typename TO>
__device__ __forceinline__ u32x4 ld_chunk_as(const TO* src) {
  if constexpr (__is_same(T, TO)) {
    return ld16(src);
  } else {
    static_assert(__is_same(TO, float) && sizeof(T) == 2, "float -> 16-bit only");
    const f32x4 a = *reinterpret_cast<const f32x4*>(src);
    const f32x4 b = *reinterpret_cast<const f32x4*>(src + 4);
    Frag<T> f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[e] = (T)a[e];
      f[4 + e] = (T)b[e];
    }
    return __builtin_bit_cast(u32x4, f);
  }
}

// Eight consecutive elements of a TO array as a fragment of T.
template <typename T, typename TO>
__device__ __forceinline__ Frag<T> ld_frag_as(const TO* src) {
  if constexpr (__is_same(T, TO)) {
    return *reinterpret_cast<const Frag<T>*>(src);
  } else {
    const f32x8 x = *reinterpret_cast<const f32x8*>(src);
    Frag<T> f;
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = (T)x[e];
    return f;
  }
}

// Workgroup id remap for the 8 XCDs of the chip: hardware hands workgroup w to
// XCD w % 8, so give each XCD a contiguous range of logical tiles (neighbours
// share K/V in that XCD's L2).  Bijective on [0, n).
__device__ __forceinline__ int xcd_remap(int w, int n) {
  const int x = w & 7, i = w >> 3;
  const int per = n >> 3, rem = n & 7;
  return x * per + (x < rem ? x : rem) + i;
}

// (batch, head) index of the g-th (batch, head) pair in the order the grid
// enumerates them: batch fastest, then head.  Consecutive logical tiles (and so
// each XCD's contiguous range of them) then mix all batches, which keeps the
// XCDs evenly loaded when batches have different valid key lengths, while the
// tiles of one (batch, head) stay together.  Bijective on [0, bh).
__device__ __forceinline__ int bh_of_group(int g, int bh, int heads) {
  const int batch = bh / heads;
  return (g % batch) * heads + g / batch;
}

}  // namespace mea
