// C ABI of the attention library: argument validation, work planning
// (query tiles, key splits, workspace carving) and kernel dispatch.  Nothing
// here allocates device memory or synchronises; every launch goes onto the
// caller's stream.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <mutex>

#include "../../include/mea.h"
#include "kernels.hpp"

// Per-row backward workspace of mea_attention_bwd_noalloc: one copy per GPU,
// allocated when the library's code object is loaded on that GPU.  In host
// code the name `scratch` is only a host-side stand-in; its device address is
// looked up per device (scratch_of_device) and only that address is used.
static __device__ __align__(256) unsigned char scratch[MEA_NOALLOC_SCRATCH_BYTES];

namespace {

using mea::BwdParams;
using mea::FwdParams;

constexpr int64_t kMaxSeq = (int64_t)1 << 31;  // n_q, n_k must stay below 2^31

bool mul_ok(int64_t a, int64_t b, int64_t* out) {
  if (a < 0 || b < 0) return false;
  if (a != 0 && b > INT64_MAX / a) return false;
  *out = a * b;
  return true;
}

// Head dimension of v and o (d_v = 0 means d).
int64_t dv_of(const mea_problem* p) { return p->d_v ? p->d_v : p->d; }

// Shape, dtype and scale checks shared by every entry point.
mea_status check_problem(const mea_problem* p) {
  if (!p) return MEA_ERR_INVALID_ARG;
  if (p->batch < 1 || p->heads < 1 || p->n_q < 1 || p->n_k < 1 || p->d < 1)
    return MEA_ERR_INVALID_ARG;
  if (p->n_q >= kMaxSeq || p->n_k >= kMaxSeq) return MEA_ERR_INVALID_ARG;
  if (p->causal != 0 && p->causal != 1) return MEA_ERR_INVALID_ARG;
  if (p->out_f32 != 0 && p->out_f32 != 1) return MEA_ERR_INVALID_ARG;
  if (!(p->scale > 0.0f) || !isfinite(p->scale)) return MEA_ERR_INVALID_ARG;
  if (p->kv_len && ((uintptr_t)p->kv_len & 3u)) return MEA_ERR_INVALID_ARG;
  if (p->d_v < 0) return MEA_ERR_INVALID_ARG;
  const int64_t dmax = p->d > dv_of(p) ? p->d : dv_of(p);
  int64_t bh, nq_d, nk_d, tot;
  if (!mul_ok(p->batch, p->heads, &bh) || bh >= kMaxSeq) return MEA_ERR_INVALID_ARG;
  if (!mul_ok(p->n_q, dmax, &nq_d) || !mul_ok(p->n_k, dmax, &nk_d)) return MEA_ERR_INVALID_ARG;
  if (!mul_ok(bh, nq_d, &tot) || !mul_ok(bh, nk_d, &tot)) return MEA_ERR_INVALID_ARG;
  if (!mul_ok(bh, p->n_q * 4, &tot)) return MEA_ERR_INVALID_ARG;
  if (p->d != 64 && p->d != 128) return MEA_ERR_UNSUPPORTED;
  if (dv_of(p) != 64 && dv_of(p) != 128) return MEA_ERR_UNSUPPORTED;
  if (p->dtype != MEA_F32 && p->dtype != MEA_F16 && p->dtype != MEA_BF16) return MEA_ERR_UNSUPPORTED;
  return MEA_OK;
}

// Strides of a tensor of n rows of w features: given, or contiguous [B, H, n, w].
mea::TensorStrides strides_of(const mea_problem* p, const mea_tensor_strides* given, int64_t n, int64_t w) {
  if (given) return {given->batch, given->head, given->row};
  return {p->heads * n * w, n * w, w};
}

// Validation of one tensor's strides (see mea.h); w = features per row.
bool strides_ok(const mea_problem* p, const mea::TensorStrides& s, int64_t n, bool output, size_t elem,
                int64_t w) {
  const int64_t align = 16 / (int64_t)elem;
  if (s.b < 0 || s.h < 0 || s.r < w || s.r >= ((int64_t)1 << 24)) return false;
  if (output && (s.b == 0 || s.h == 0)) return false;
  if (s.b % align || s.h % align || s.r % align) return false;
  int64_t a, b, c, tot;
  if (!mul_ok(p->batch - 1, s.b, &a) || !mul_ok(p->heads - 1, s.h, &b) || !mul_ok(n - 1, s.r, &c)) return false;
  if (__builtin_add_overflow(a, b, &tot) || __builtin_add_overflow(tot, c, &tot) ||
      __builtin_add_overflow(tot, w, &tot))
    return false;
  return true;
}

size_t elem_size(int32_t dtype) { return dtype == MEA_F32 ? 4 : 2; }

// Whether o and do are float32 (float32 inputs, or 16-bit inputs with out_f32).
bool out_is_f32(const mea_problem* p) { return p->dtype == MEA_F32 || p->out_f32 != 0; }

bool aligned16(const void* ptr) { return ((uintptr_t)ptr & 15u) == 0; }
bool dev_ptr_ok(const void* ptr) { return ptr != nullptr && aligned16(ptr); }

struct FwdPlan {
  int bq, bk;
  int64_t n_qtiles;
  int n_splits;
  int64_t keys_per_split;
  size_t workspace;
};

void fwd_tiles(int dtype, int64_t d, int64_t dv, bool causal, int64_t n_q, int64_t bh, int* bq, int* bk) {
  if (dtype == MEA_F32) {
    *bq = mea::FwdShape<float, 64>::BQ;
    *bk = mea::FwdShape<float, 64>::BK;
  } else if (d == 64 && dv == 64) {
    *bq = mea::FwdShape<__bf16, 64>::BQ == 512 ? mea::fwd64_bq(n_q, bh, causal) : mea::FwdShape<__bf16, 64>::BQ;
    *bk = mea::FwdShape<__bf16, 64>::BK;
  } else if (d == 128 && dv == 128) {
    *bq = mea::FwdShape<__bf16, 128>::BQ == 256 ? mea::fwd128_bq(n_q, causal) : mea::FwdShape<__bf16, 128>::BQ;
    *bk = mea::FwdShape<__bf16, 128>::BK;
  } else {  // d_v != d: the 4-wave kernel
    *bq = mea::kFwdBq4wave128;
    *bk = mea::FwdShape<__bf16, 128>::BK;
  }
}

// Grid plan.  The chip has 256 CUs; when the query tiles alone give too few
// workgroups, the keys are split so that each split's summary is combined
// afterwards (Section 4 combine).
// Decode plan: one wave per key range; ranges of at least 4 key tiles, about
// MEA_DECODE_TARGET_WG workgroups in all, at most 1024 ranges per (batch,
// head).  1024 workgroups are one round of four per CU (the LDS ring allows
// four): 2.5 % faster than two rounds at 8 x 16 heads, 65536 keys.
#ifndef MEA_DECODE_TARGET_WG
#define MEA_DECODE_TARGET_WG 1024
#endif
FwdPlan plan_decode(const mea_problem* p) {
  FwdPlan pl;
  pl.bq = 64;
  pl.bk = mea::fwd_decode_tile((int)p->d);
  pl.n_qtiles = 1;
  const int64_t bh = p->batch * p->heads;
  const int64_t n_keys = p->causal && p->n_k > p->n_q ? p->n_q : p->n_k;
  const int64_t k_tiles = (n_keys + pl.bk - 1) / pl.bk;
  int64_t splits = (MEA_DECODE_TARGET_WG + bh - 1) / bh;
  if (splits > k_tiles / 4) splits = k_tiles / 4;
  if (splits > 1024) splits = 1024;
  if (splits < 1) splits = 1;
  const int64_t tiles_per_split = (k_tiles + splits - 1) / splits;
  pl.keys_per_split = tiles_per_split * pl.bk;
  pl.n_splits = (int)((n_keys + pl.keys_per_split - 1) / pl.keys_per_split);
  pl.workspace = 0;
  if (pl.n_splits > 1) {
    const size_t rows = (size_t)pl.n_splits * (size_t)bh * (size_t)p->n_q;
    const size_t stage = mea::combine_stage_floats(pl.n_splits, bh * p->n_q, dv_of(p));
    pl.workspace = rows * (size_t)dv_of(p) * 4 + 2 * rows * 4 + 256 + (stage ? stage * 4 + 256 : 0);
  }
  return pl;
}

FwdPlan plan_fwd(const mea_problem* p) {
  if (mea::fwd_uses_decode((int)p->dtype, (int)p->d, (int)dv_of(p), p->n_q)) return plan_decode(p);
  FwdPlan pl;
  const int64_t bh = p->batch * p->heads;
  fwd_tiles(p->dtype, p->d, dv_of(p), p->causal != 0, p->n_q, bh, &pl.bq, &pl.bk);
  pl.n_qtiles = (p->n_q + pl.bq - 1) / pl.bq;
  const int64_t k_tiles = (p->n_k + pl.bk - 1) / pl.bk;
  const int64_t base = bh * pl.n_qtiles;
  int64_t splits = 1;
  // Whole rounds of workgroups: 1024 (four per CU) for the kernels that fit
  // one or two per CU, one round of MEA_T64_FWD_OCC per CU for the 16-bit
  // d = 64 4-wave kernel (three: 768 workgroups measured 2-12 % faster than
  // 1024 on 65-256 queries against 32768-262144 keys, and the same as 1536).
  const bool four_wave64 = pl.bq == 128 && p->dtype != MEA_F32 && p->d == 64 && dv_of(p) == 64;
  const int64_t kTargetWorkgroups = four_wave64 ? 256 * MEA_T64_FWD_OCC : 1024;
  const int64_t kMinTilesPerSplit = 16;
  if (base < 512 && k_tiles >= 2 * kMinTilesPerSplit) {
    splits = (kTargetWorkgroups + base - 1) / base;
    const int64_t max_splits = k_tiles / kMinTilesPerSplit;
    if (splits > max_splits) splits = max_splits;
    if (splits > 64) splits = 64;
    if (splits < 1) splits = 1;
  }
  const int64_t tiles_per_split = (k_tiles + splits - 1) / splits;
  pl.keys_per_split = tiles_per_split * pl.bk;
  pl.n_splits = (int)((p->n_k + pl.keys_per_split - 1) / pl.keys_per_split);
  pl.workspace = 0;
  if (pl.n_splits > 1) {
    const size_t rows = (size_t)pl.n_splits * (size_t)bh * (size_t)p->n_q;
    const size_t stage = mea::combine_stage_floats(pl.n_splits, bh * p->n_q, dv_of(p));
    pl.workspace = rows * (size_t)dv_of(p) * 4 + 2 * rows * 4 + 256 + (stage ? stage * 4 + 256 : 0);
  }
  return pl;
}

int64_t bwd_row_pad(int64_t n_q) { return (n_q + mea::kBwdRowPad - 1) / mea::kBwdRowPad * mea::kBwdRowPad; }

// Bytes of one per-row backward array of `elem` bytes per row, rounded to 256.
size_t bwd_row_array_bytes(const mea_problem* p, size_t elem) {
  const size_t b = (size_t)p->batch * (size_t)p->heads * (size_t)bwd_row_pad(p->n_q) * elem;
  return (b + 255) / 256 * 256;
}

// Whether the backward keeps a 16-bit copy of a float32 dO (16-bit inputs,
// float32 outputs) so that the kernels of 16-bit outputs run: `allow` is false
// for the allocation-free entry point, whose scratch holds the per-row values
// only (those problems then run the kernels that convert dO while staging it;
// the results are the same).
bool bwd_do16(const mea_problem* p, bool allow) { return allow && p->dtype != MEA_F32 && p->out_f32 != 0; }

bool bwd_records(const mea_problem* p, bool allow_do16) {
  const bool f32_do = p->dtype != MEA_F32 && p->out_f32 != 0 && !bwd_do16(p, allow_do16);
  return mea::bwd_uses_row_records((int)p->dtype, (int)p->d, (int)dv_of(p), f32_do, p->causal != 0, p->n_q);
}

size_t bwd_do16_bytes(const mea_problem* p) {
  const size_t b = (size_t)p->batch * (size_t)p->heads * (size_t)p->n_q * (size_t)dv_of(p) * 2;
  return (b + 255) / 256 * 256;
}

size_t bwd_workspace(const mea_problem* p, bool allow_do16) {
  // One 16-byte record per padded row (two-group kernels), or s_init and
  // dp_init as [B*H, n_q_pad] float32 arrays; then the 16-bit dO copy, if
  // any; 256-byte aligned.
  const size_t rows = bwd_records(p, allow_do16) ? bwd_row_array_bytes(p, 16) : 2 * bwd_row_array_bytes(p, 4);
  return rows + (bwd_do16(p, allow_do16) ? bwd_do16_bytes(p) : 0) + 256;
}

float* align256(void* base, size_t off) {
  uintptr_t a = (uintptr_t)base + off;
  a = (a + 255u) & ~(uintptr_t)255u;
  return reinterpret_cast<float*>(a);
}

constexpr float kLog2e = 1.4426950408889634f;

// Device address of `scratch` on the current device, looked up once per
// device (hipGetSymbolAddress with that device current) and cached.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

mea_status scratch_of_device(hipStream_t stream, void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return MEA_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return MEA_ERR_UNSUPPORTED;
  if (stream) {
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice(stream, &sdev) != hipSuccess) return MEA_ERR_HIP;
    if (sdev != dev) return MEA_ERR_INVALID_ARG;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return MEA_ERR_HIP;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return MEA_OK;
}

// Checks of the backward's pointers (before anything is launched).
mea_status check_bwd_pointers(const mea_problem* p, const void* q, const void* k, const void* v,
                              const void* o, const void* o_lo, const void* d_o, const float* lse,
                              const void* dq, const void* dk, const void* dv) {
  if (!dev_ptr_ok(q) || !dev_ptr_ok(k) || !dev_ptr_ok(v) || !dev_ptr_ok(o) || !dev_ptr_ok(d_o) ||
      !dev_ptr_ok(lse))
    return MEA_ERR_INVALID_ARG;
  if (o_lo && (!aligned16(o_lo) || out_is_f32(p))) return MEA_ERR_INVALID_ARG;
  // dq may be NULL (dQ skipped); dk and dv are both given or both NULL.
  if ((dq && !aligned16(dq)) || (dk && !aligned16(dk)) || (dv && !aligned16(dv)))
    return MEA_ERR_INVALID_ARG;
  if ((dk == nullptr) != (dv == nullptr)) return MEA_ERR_INVALID_ARG;
  if (!dq && !dk) return MEA_ERR_INVALID_ARG;
  return MEA_OK;
}

mea_status bwd_launch(const mea_problem* p, const void* q, const void* k, const void* v, const void* o,
                      const void* o_lo, const void* d_o, const float* lse, void* dq, void* dk, void* dv,
                      void* workspace, bool allow_do16, hipStream_t stream);

}  // namespace

extern "C" {

const char* mea_status_string(mea_status s) {
  // A C caller may pass any int: read the raw value instead of loading an
  // enumeration value that may lie outside its range.
  int code = 0;
  memcpy(&code, &s, sizeof(code) < sizeof(s) ? sizeof(code) : sizeof(s));
  switch (code) {
    case MEA_OK: return "ok";
    case MEA_ERR_INVALID_ARG: return "invalid argument";
    case MEA_ERR_UNSUPPORTED: return "unsupported head dimension or dtype";
    case MEA_ERR_WORKSPACE: return "workspace missing or too small";
    case MEA_ERR_HIP: return "HIP runtime error at launch";
    case MEA_ERR_SCRATCH: return "problem needs more workspace than the static scratch of the allocation-free entry point (MEA_NOALLOC_SCRATCH_BYTES)";
  }
  return "unknown status";
}

mea_status mea_attention_fwd_workspace_size(const mea_problem* p, size_t* bytes) {
  const mea_status st = check_problem(p);
  if (st != MEA_OK) return st;
  if (!bytes) return MEA_ERR_INVALID_ARG;
  *bytes = plan_fwd(p).workspace;
  return MEA_OK;
}

mea_status mea_attention_bwd_workspace_size(const mea_problem* p, size_t* bytes) {
  const mea_status st = check_problem(p);
  if (st != MEA_OK) return st;
  if (!bytes) return MEA_ERR_INVALID_ARG;
  *bytes = bwd_workspace(p, true);
  return MEA_OK;
}

mea_status mea_attention_fwd(const mea_problem* p, const void* q, const void* k, const void* v,
                             void* o, float* lse, void* o_lo, void* workspace, size_t workspace_bytes,
                             hipStream_t stream) {
  const mea_status st = check_problem(p);
  if (st != MEA_OK) return st;
  if (!dev_ptr_ok(q) || !dev_ptr_ok(k) || !dev_ptr_ok(v) || !dev_ptr_ok(o))
    return MEA_ERR_INVALID_ARG;
  if (lse && !aligned16(lse)) return MEA_ERR_INVALID_ARG;
  if (o_lo && (!aligned16(o_lo) || out_is_f32(p))) return MEA_ERR_INVALID_ARG;
  const FwdPlan pl = plan_fwd(p);
  if (pl.workspace > 0 && (!workspace || workspace_bytes < pl.workspace)) return MEA_ERR_WORKSPACE;

  FwdParams fp = {};
  fp.q = q;
  fp.k = k;
  fp.v = v;
  fp.o = o;
  fp.lse = lse;
  fp.o_lo = o_lo;
  fp.kv_len = p->kv_len;
  fp.n_q = p->n_q;
  fp.n_k = p->n_k;
  fp.keys_per_split = pl.keys_per_split;
  fp.bh = (int)(p->batch * p->heads);
  fp.n_qtiles = (int)pl.n_qtiles;
  fp.n_splits = pl.n_splits;
  fp.scale = p->scale;
  fp.scale_log2 = p->scale * kLog2e;
  fp.heads = (int)p->heads;
  {
    const mea_strides* st_ = p->strides;
    const size_t e = elem_size(p->dtype), eo = p->out_f32 && p->dtype != MEA_F32 ? 4 : e;
    const int64_t d = p->d, dv = dv_of(p);
    fp.sq = strides_of(p, st_ ? &st_->q : nullptr, p->n_q, d);
    fp.sk = strides_of(p, st_ ? &st_->k : nullptr, p->n_k, d);
    fp.sv = strides_of(p, st_ ? &st_->v : nullptr, p->n_k, dv);
    fp.so = strides_of(p, st_ ? &st_->o : nullptr, p->n_q, dv);
    if (!strides_ok(p, fp.sq, p->n_q, false, e, d) || !strides_ok(p, fp.sk, p->n_k, false, e, d) ||
        !strides_ok(p, fp.sv, p->n_k, false, e, dv) || !strides_ok(p, fp.so, p->n_q, true, eo, dv))
      return MEA_ERR_INVALID_ARG;
  }
  if (pl.n_splits > 1) {
    const size_t rows = (size_t)pl.n_splits * (size_t)fp.bh * (size_t)p->n_q;
    fp.part_o = align256(workspace, 0);
    fp.part_m = fp.part_o + rows * (size_t)dv_of(p);
    fp.part_l = fp.part_m + rows;
    const int64_t rows1 = (int64_t)fp.bh * p->n_q;
    if (mea::combine_stage_floats(pl.n_splits, rows1, dv_of(p)) > 0) {
      const size_t r2 = (size_t)((pl.n_splits + mea::kCombineGroup - 1) / mea::kCombineGroup) * (size_t)rows1;
      fp.part2_o = align256(fp.part_l + rows, 0);
      fp.part2_m = fp.part2_o + r2 * (size_t)dv_of(p);
      fp.part2_l = fp.part2_m + r2;
    }
  }
  const int64_t grid = (int64_t)fp.n_qtiles * fp.bh * fp.n_splits;
  if (grid >= ((int64_t)1 << 31)) return MEA_ERR_INVALID_ARG;
  const hipError_t e = mea::launch_fwd(fp, p->dtype, (int)p->d, (int)dv_of(p), p->causal != 0,
                                       p->out_f32 != 0, stream);
  return e == hipSuccess ? MEA_OK : MEA_ERR_HIP;
}

mea_status mea_attention_bwd(const mea_problem* p, const void* q, const void* k, const void* v,
                             const void* o, const void* o_lo, const void* d_o, const float* lse, void* dq,
                             void* dk, void* dv, void* workspace, size_t workspace_bytes,
                             hipStream_t stream) {
  mea_status st = check_problem(p);
  if (st != MEA_OK) return st;
  st = check_bwd_pointers(p, q, k, v, o, o_lo, d_o, lse, dq, dk, dv);
  if (st != MEA_OK) return st;
  const size_t need = bwd_workspace(p, true);
  if (!workspace || workspace_bytes < need) return MEA_ERR_WORKSPACE;
  return bwd_launch(p, q, k, v, o, o_lo, d_o, lse, dq, dk, dv, workspace, true, stream);
}

mea_status mea_attention_bwd_noalloc(const mea_problem* p, const void* q, const void* k, const void* v,
                                     const void* o, const void* o_lo, const void* d_o, const float* lse,
                                     void* dq, void* dk, void* dv, hipStream_t stream) {
  mea_status st = check_problem(p);
  if (st != MEA_OK) return st;
  st = check_bwd_pointers(p, q, k, v, o, o_lo, d_o, lse, dq, dk, dv);
  if (st != MEA_OK) return st;
  if (bwd_workspace(p, false) > MEA_NOALLOC_SCRATCH_BYTES) return MEA_ERR_SCRATCH;
  void* ws = nullptr;
  st = scratch_of_device(stream, &ws);
  if (st != MEA_OK) return st;
  return bwd_launch(p, q, k, v, o, o_lo, d_o, lse, dq, dk, dv, ws, false, stream);
}

}  // extern "C"

namespace {

// The backward after validation: kernel arguments, stride checks, launches.
// `workspace` holds at least bwd_workspace(p, allow_do16) bytes.
mea_status bwd_launch(const mea_problem* p, const void* q, const void* k, const void* v, const void* o,
                      const void* o_lo, const void* d_o, const float* lse, void* dq, void* dk, void* dv,
                      void* workspace, bool allow_do16, hipStream_t stream) {
  BwdParams bp = {};
  bp.q = q;
  bp.k = k;
  bp.v = v;
  bp.o = o;
  bp.o_lo = o_lo;
  bp.d_o = d_o;
  bp.lse = lse;
  bp.dq = dq;
  bp.dk = dk;
  bp.dv = dv;
  bp.n_q_pad = bwd_row_pad(p->n_q);
  const bool rec = bwd_records(p, allow_do16);
  if (rec) {
    bp.row_rec = reinterpret_cast<uint4*>(align256(workspace, 0));
  } else {
    bp.s_init = align256(workspace, 0);
    bp.dp_init = bp.s_init + bwd_row_array_bytes(p, 4) / 4;
  }
  if (bwd_do16(p, allow_do16))
    bp.do16 = align256(workspace, rec ? bwd_row_array_bytes(p, 16) : 2 * bwd_row_array_bytes(p, 4));
  bp.kv_len = p->kv_len;
  bp.n_q = p->n_q;
  bp.n_k = p->n_k;
  bp.bh = (int)(p->batch * p->heads);
  bp.scale = p->scale;
  bp.scale_log2 = p->scale * kLog2e;
  bp.heads = (int)p->heads;
  {
    const mea_strides* st_ = p->strides;
    const size_t e = elem_size(p->dtype), eo = p->out_f32 && p->dtype != MEA_F32 ? 4 : e;
    const int64_t d = p->d, dvw = dv_of(p);
    bp.sq = strides_of(p, st_ ? &st_->q : nullptr, p->n_q, d);
    bp.sk = strides_of(p, st_ ? &st_->k : nullptr, p->n_k, d);
    bp.sv = strides_of(p, st_ ? &st_->v : nullptr, p->n_k, dvw);
    bp.so = strides_of(p, st_ ? &st_->o : nullptr, p->n_q, dvw);
    bp.sdo = strides_of(p, st_ ? &st_->d_o : nullptr, p->n_q, dvw);
    bp.sdq = strides_of(p, st_ ? &st_->dq : nullptr, p->n_q, d);
    bp.sdk = strides_of(p, st_ ? &st_->dk : nullptr, p->n_k, d);
    bp.sdv = strides_of(p, st_ ? &st_->dv : nullptr, p->n_k, dvw);
    if (!strides_ok(p, bp.sq, p->n_q, false, e, d) || !strides_ok(p, bp.sk, p->n_k, false, e, d) ||
        !strides_ok(p, bp.sv, p->n_k, false, e, dvw) || !strides_ok(p, bp.so, p->n_q, false, eo, dvw) ||
        !strides_ok(p, bp.sdo, p->n_q, false, eo, dvw) || (dq && !strides_ok(p, bp.sdq, p->n_q, true, e, d)) ||
        (dk && (!strides_ok(p, bp.sdk, p->n_k, true, e, d) || !strides_ok(p, bp.sdv, p->n_k, true, e, dvw))))
      return MEA_ERR_INVALID_ARG;
  }
  const hipError_t e = mea::launch_bwd(bp, p->dtype, (int)p->d, (int)dv_of(p), p->causal != 0,
                                       p->out_f32 != 0, stream);
  if (e == hipErrorNotSupported) return MEA_ERR_UNSUPPORTED;
  return e == hipSuccess ? MEA_OK : MEA_ERR_HIP;
}

}  // namespace
