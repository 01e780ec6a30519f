// Host-side interface between the C ABI (api.hip) and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mea {

// Element strides of one [B, H, n, d] tensor (batch, head, row); features
// are contiguous.  Row 0 of (batch, head) bh starts at head_base(s, bh, H).
struct TensorStrides {
  int64_t b, h, r;
};
__host__ __device__ inline int64_t head_base(const TensorStrides& s, int bh, int heads) {
  return (int64_t)(bh / heads) * s.b + (int64_t)(bh % heads) * s.h;
}

// Keys visible to every query of (batch, head) bh: the batch's valid key
// length from kv_len (device array [B], clamped to [0, n_k]) or all n_k.
// Keys from there to n_k are masked like keys past the end; they stay
// readable memory, so loads are bounded by n_k.
__device__ inline int64_t valid_keys(const int* kv_len, int bh, int heads, int64_t n_k) {
  if (kv_len == nullptr) return n_k;
  const int64_t l = kv_len[bh / heads];
  return l < 0 ? 0 : (l > n_k ? n_k : l);
}

// Arguments of the forward kernels (passed by value).
struct FwdParams {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  float* lse;     // [B*H, n_q] or null
  void* o_lo;     // 16-bit o only: rounding residual of o, contiguous [B*H, n_q, DV], or null
  float* part_o;  // split partials [S, B*H, n_q, D] (n_splits > 1)
  float* part_m;  // [S, B*H, n_q]
  float* part_l;  // [S, B*H, n_q]
  // Second partial buffer for the staged combine (n_splits > kCombineGroup):
  // ceil(S / kCombineGroup) splits in the same layout.
  float* part2_o;
  float* part2_m;
  float* part2_l;
  const int* kv_len;  // [B] valid keys per batch, or null (all n_k)
  int64_t n_q;
  int64_t n_k;
  int64_t keys_per_split;  // multiple of the key tile
  int bh;                  // B * H
  int n_qtiles;
  int n_splits;
  float scale;       // score scale
  float scale_log2;  // scale * log2(e)
  int heads;         // H (bh = b * H + h)
  TensorStrides sq, sk, sv, so;
};

// The summaries of more than kCombineGroup key ranges are combined in stages
// of kCombineGroup ranges each (Section 4's combine applied as a tree), so
// that the work stays parallel when there are few rows and many ranges.
constexpr int kCombineGroup = 16;

// Lazy reference maximum of the forward kernels (Section 3's running maximum,
// raised lazily): a tile raises the reference only when one of its scores
// exceeds it by more than this many powers of two, so weights stay <= 2^8 and
// the running numerator and denominator are rescaled only on such tiles.
constexpr float kRescaleSlack = 8.0f;
constexpr float kRescaleBound = 256.0f;  // 2^kRescaleSlack

// Floats of the second partial buffer (0 when the combine is one stage).
inline size_t combine_stage_floats(int64_t n_splits, int64_t rows, int64_t d) {
  if (n_splits <= kCombineGroup) return 0;
  const int64_t s1 = (n_splits + kCombineGroup - 1) / kCombineGroup;
  return (size_t)s1 * (size_t)rows * (size_t)(d + 2);
}

// Arguments of the backward kernels.
struct BwdParams {
  const void* q;
  const void* k;
  const void* v;
  const void* o;
  const void* o_lo;  // residual of a 16-bit o (contiguous [B*H, n_q, DV]) or null
  const void* d_o;
  const float* lse;
  void* dq;
  void* dk;
  void* dv;
  // Per-row initial values of the score and dP accumulators, written by the
  // preprocess kernel: s_init = -lse / scale (so that P = 2^(c * (S + s_init)),
  // c = scale * log2 e) and dp_init = -D with D_i = dO_i . O_i (so that
  // dS = P * (dP + dp_init)).  Rows n_q .. n_q_pad - 1 contribute nothing.
  // The two-group kernels (16-bit inputs and outputs, d = 64) take them as
  // one 16-byte record per row, eight bf16 values {s_hi, s_mid, s_lo, 0,
  // d_hi, d_mid, d_lo, 0} whose three parts sum to s_init and dp_init in
  // float32 (padding rows: s = -2^100, d = 0), so that one bf16 MFMA against
  // a constant operand puts them into the accumulators; the other kernels
  // take [B*H, n_q_pad] float32 arrays (padding rows -inf and 0).
  float* s_init;
  float* dp_init;
  uint4* row_rec;
  // 16-bit inputs with float32 o and dO: dO rounded to the input dtype
  // (contiguous [B*H, n_q, DV]), written by the preprocess, so that the
  // dK/dV and dQ kernels of 16-bit outputs run on it; or null.
  void* do16;
  const int* kv_len;  // [B] valid keys per batch, or null (all n_k)
  int64_t n_q_pad;  // n_q rounded up to kBwdRowPad
  int64_t n_q;
  int64_t n_k;
  int bh;
  int n_qtiles;  // query tiles of the dQ kernel
  int n_ktiles;  // key tiles of the dK/dV kernel
  float scale;
  float scale_log2;
  int heads;  // H (bh = b * H + h)
  TensorStrides sq, sk, sv, so, sdo, sdq, sdk, sdv;
};

// Row padding of the backward's per-row arrays (a multiple of every query
// tile the backward kernels stage).
constexpr int kBwdRowPad = 64;

// Whether the backward runs the two-group kernels, which take the per-row
// values as 16-byte records; every other backward takes them as two float32
// arrays.  The host's workspace layout and the kernels' choice both come from
// this one predicate.  Causal problems of up to MEA_T64_BWD_CAUSAL_SMALL
// queries run the 4-wave kernels: measured on causal bf16 d = 64 problems,
// n = 1024-2048 (128-256 heads) took 5-13 % less time with them; at 3072 the
// two kinds tie, and from 4096 queries on the two-group kernels take 3-12 %
// less (6-7 % more before their plain tiles dropped the mask).  Unmasked
// problems of up to MEA_T64_BWD_SHORT queries run them too (the two-group dQ
// kernel's 256-query tiles are mostly padding there): bf16 d = 64, two-group /
// 4-wave, dK/dV + dQ: 2.796 / 2.293 ms at 8x16 heads, 65 queries, 65536
// keys; 3.123 / 2.886 at 256; 4.543 / 4.563 at 512; 0.226 / 0.180 at 4x32
// heads, 128 queries, 4096 keys; 0.343 / 0.324 at 512; 0.550 / 0.552 at
// 1024; 0.292 / 0.303 at 4x16x2048^2.  The two kinds give bitwise the same
// gradients.
#ifndef MEA_T64_BWD_CAUSAL_SMALL
#define MEA_T64_BWD_CAUSAL_SMALL 2048
#endif
#ifndef MEA_T64_BWD_SHORT
#define MEA_T64_BWD_SHORT 512
#endif
// Whether the two-group backward kernels exist for these types and head
// dimensions (whatever the problem's shape).
constexpr bool bwd_two_group_exists(bool is16, int d, int dv, bool same_out_dtype) {
  return is16 && d == 64 && dv == 64 && same_out_dtype;
}
constexpr bool bwd_two_group(bool is16, int d, int dv, bool same_out_dtype, bool causal, int64_t n_q) {
  return bwd_two_group_exists(is16, d, dv, same_out_dtype) && !(causal && n_q <= MEA_T64_BWD_CAUSAL_SMALL) &&
         !(!causal && n_q <= MEA_T64_BWD_SHORT);
}
// dtype: 0 float32, 1 fp16, 2 bf16; d and dv the head dimensions of q, k and
// of v, o.
inline bool bwd_uses_row_records(int dtype, int d, int dv, bool out_f32, bool causal, int64_t n_q) {
  return bwd_two_group(dtype != 0, d, dv, !out_f32, causal, n_q);
}

// Tile shapes per (element type, head dimension); shared by the host plan
// and the kernel instantiations.
// 16-bit d = 64 forward: BQ = 512 selects the two-group ping-pong kernel
// (8 waves); otherwise the 4-wave kernel runs with QT = BQ / 128 query
// sub-tiles per wave and MEA_T64_FWD_OCC workgroups per CU.
#ifndef MEA_T64_FWD_BQ
#define MEA_T64_FWD_BQ 512
#endif
// Three workgroups per CU (166 registers, no spills) measured 4-10 % faster
// than two on the causal problems this kernel runs (4x32x4096, 8x16x2048,
// 16x16x1024).
#ifndef MEA_T64_FWD_OCC
#define MEA_T64_FWD_OCC 3
#endif
template <typename T, int D> struct FwdShape;
template <> struct FwdShape<__bf16, 64> {
  static constexpr int BQ = MEA_T64_FWD_BQ, QT = BQ == 512 ? 2 : BQ / 128, BK = 64, OCC = MEA_T64_FWD_OCC;
};
// 16-bit d = d_v = 64 causal forward: the two-group kernel (512-query
// workgroups, returns 512) for problems of more than MEA_T64_FWD_CAUSAL_SMALL
// queries with at least MEA_T64_FWD_CAUSAL_MIN_PAIRS (batch x heads x n_q^2)
// query-key pairs and at least MEA_T64_FWD_CAUSAL_MIN_WGS such workgroups,
// else the 4-wave kernel with 128-query workgroups (128).  A 512-query
// workgroup spends 8 key tiles on the diagonal, half of that work masked,
// which short sequences do not amortise, and a small grid of such workgroups
// (a few hundred, for 256 CUs) balances poorly.  Measured on causal bf16
// problems, the 4-wave kernel at three workgroups per CU against the
// two-group kernel: 2-3 % faster at 4x32x4608 and 8x16x6144, 5 % at
// 1x4x32768 (256 two-group workgroups), and faster at every n <= 4096; the
// two-group kernel 3.5, 8 and 18 % faster at 4x32x8192, 2x16x12288 and
// 1x16x16384.  Host plan and launch both use this.
#ifndef MEA_T64_FWD_CAUSAL_SMALL
#define MEA_T64_FWD_CAUSAL_SMALL 6144
#endif
#ifndef MEA_T64_FWD_CAUSAL_MIN_PAIRS
#define MEA_T64_FWD_CAUSAL_MIN_PAIRS 2.5e9
#endif
#ifndef MEA_T64_FWD_CAUSAL_MIN_WGS
#define MEA_T64_FWD_CAUSAL_MIN_WGS 384
#endif
inline int fwd_causal64_bq(int64_t n_q, int64_t bh) {
  const bool big = n_q > MEA_T64_FWD_CAUSAL_SMALL &&
                   (double)bh * (double)n_q * (double)n_q >= (double)MEA_T64_FWD_CAUSAL_MIN_PAIRS &&
                   bh * ((n_q + 511) / 512) >= MEA_T64_FWD_CAUSAL_MIN_WGS;
  return big ? 512 : 128;
}
// 16-bit d = d_v forward without the causal mask: the 4-wave kernel with
// 128-query workgroups when the two-group kernel's one query tile (BQ_pp =
// 512 queries at d = 64, 256 at d = 128) would be at least half padding,
// else the two-group kernel.  Measured (bf16, two-group / 4-wave): d = 64,
// 8x16 heads, 65536 keys: 0.907 / 0.497 ms at 65 queries, 1.009 / 0.797 at
// 256, 1.036 / 1.118 at 300, 1.184 / 1.532 at 512; d = 128: 1.003 / 0.781 at
// 65, 1.060 / 0.840 at 128, 1.041 / 1.361 at 160, 1.169 / 1.479 at 256.
// Above that the two kernels measured within about 10 % either way, with
// the two-group kernel ahead on the larger problems.
inline bool fwd_pp_unmasked(int64_t n_q, int bq_pp) { return 2 * n_q > bq_pp; }
// 16-bit d = d_v = 64 forward: queries per workgroup (512: the two-group
// kernel; 128: the 4-wave kernel).
inline int fwd64_bq(int64_t n_q, int64_t bh, bool causal) {
  if (causal) return fwd_causal64_bq(n_q, bh);
  return fwd_pp_unmasked(n_q, 512) ? 512 : 128;
}
// 16-bit d = 128: BQ = 256 selects the two-group kernel (8 waves of 32
// queries); 128 the 4-wave kernel.  Problems with d_v != d always run the
// 4-wave kernel with 128 queries per workgroup (kFwdBq4wave).
#ifndef MEA_T128_FWD_BQ
#define MEA_T128_FWD_BQ 256
#endif
constexpr int kFwdBq4wave128 = 128;
// 16-bit d = d_v = 128 forward: 256 (the two-group kernel) or 128 (the 4-wave
// kernel) queries per workgroup; causal problems always run the two-group
// kernel.
inline int fwd128_bq(int64_t n_q, bool causal) {
  return causal || fwd_pp_unmasked(n_q, MEA_T128_FWD_BQ) ? MEA_T128_FWD_BQ : kFwdBq4wave128;
}
template <> struct FwdShape<__bf16, 128> { static constexpr int QT = 1, BK = 64, BQ = MEA_T128_FWD_BQ, OCC = 2; };
template <> struct FwdShape<_Float16, 64> {
  static constexpr int BQ = MEA_T64_FWD_BQ, QT = BQ == 512 ? 2 : BQ / 128, BK = 64, OCC = MEA_T64_FWD_OCC;
};
template <> struct FwdShape<_Float16, 128> { static constexpr int QT = 1, BK = 64, BQ = MEA_T128_FWD_BQ, OCC = 2; };
template <> struct FwdShape<float, 64> { static constexpr int QT = 1, BK = 32, BQ = 128, OCC = 2; };
template <> struct FwdShape<float, 128> { static constexpr int QT = 1, BK = 32, BQ = 128, OCC = 2; };

// dtype codes follow mea_dtype: 0 = f32, 1 = f16, 2 = bf16.
// out_f32: o (and, in the backward, do) are float32 instead of the input dtype.
// Decode-shaped forward: 16-bit inputs and at most 64 queries per (batch,
// head) run the key-streaming decode kernel (key tile fwd_decode_tile(d)).
inline bool fwd_uses_decode(int dtype, int d, int dv, int64_t n_q) { return dtype != 0 && d == dv && n_q <= 64; }
inline int fwd_decode_tile(int d) { return d == 64 ? 64 : 32; }
hipError_t launch_decode(const FwdParams& p, int dtype, int d, bool causal, bool out_f32, hipStream_t stream);
// dv: head dimension of v and o (equal to d, or the other of 64 and 128).
hipError_t launch_fwd(const FwdParams& p, int dtype, int d, int dv, bool causal, bool out_f32,
                      hipStream_t stream);
hipError_t launch_bwd(const BwdParams& p, int dtype, int d, int dv, bool causal, bool out_f32,
                      hipStream_t stream);

}  // namespace mea
