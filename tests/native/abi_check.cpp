// Native driver of the C ABI's host code for the sanitizer build (test
// infrastructure).  The kernel launchers are recording stubs
// (launch_stubs.cpp), so nothing runs on a GPU: every call either fails
// validation or reaches a stub, whose recorded arguments are checked here --
// the key-split plan covers every key exactly once, the workspace regions the
// entry point carves lie inside the caller's buffer and do not overlap, and
// sizes near the int64 limits are rejected instead of overflowing.  Built
// with -fsanitize=address,undefined.  Exit status = number of failures.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "../../include/mea.h"
#include "../../paper_2112_05682_amd/csrc/kernels.hpp"

namespace mea {
extern FwdParams g_last_fwd;
extern BwdParams g_last_bwd;
extern int g_fwd_calls, g_bwd_calls;
}  // namespace mea

static int failures = 0;
#define CHECK(cond, ...)                                   \
  do {                                                     \
    if (!(cond)) {                                         \
      fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
      fprintf(stderr, __VA_ARGS__);                        \
      fprintf(stderr, "\n");                               \
      ++failures;                                          \
    }                                                      \
  } while (0)

// Fake, 256-byte aligned device addresses: the stubs never dereference them.
static char* const WS = reinterpret_cast<char*>(uintptr_t(1) << 40);
static void* const P = reinterpret_cast<void*>(uintptr_t(1) << 36);

static mea_problem prob(int64_t B, int64_t H, int64_t nq, int64_t nk, int64_t d, int dtype, int causal,
                        int64_t dv = 0, int out_f32 = 0) {
  mea_problem p;
  memset(&p, 0, sizeof(p));
  p.batch = B;
  p.heads = H;
  p.n_q = nq;
  p.n_k = nk;
  p.d = d;
  p.dtype = dtype;
  p.causal = causal;
  p.scale = 0.125f;
  p.out_f32 = out_f32;
  p.d_v = dv;
  return p;
}

static bool inside(const void* a, size_t bytes, const char* base, size_t total) {
  const char* c = static_cast<const char*>(a);
  return c >= base && c + bytes <= base + total;
}
static bool disjoint(const void* a, size_t na, const void* b, size_t nb) {
  const char *x = static_cast<const char*>(a), *y = static_cast<const char*>(b);
  return x + na <= y || y + nb <= x;
}

static void check_fwd_plan(int64_t B, int64_t H, int64_t nq, int64_t nk, int64_t d, int dtype, int causal) {
  mea_problem p = prob(B, H, nq, nk, d, dtype, causal);
  size_t need = 0;
  CHECK(mea_attention_fwd_workspace_size(&p, &need) == MEA_OK, "fwd ws size");
  const int before = mea::g_fwd_calls;
  const mea_status st = mea_attention_fwd(&p, P, P, P, P, static_cast<float*>(P), nullptr,
                                          need ? WS : nullptr, need, nullptr);
  CHECK(st == MEA_OK && mea::g_fwd_calls == before + 1, "fwd call %d", (int)st);
  const mea::FwdParams& f = mea::g_last_fwd;
  if (dtype != MEA_F32 && nq > 64) {
    // The 16-bit plan tiles the queries as the kernel it picks.
    const int64_t bq = d == 64 ? mea::fwd64_bq(nq, B * H, causal) : mea::fwd128_bq(nq, causal);
    CHECK(f.n_qtiles == (nq + bq - 1) / bq, "query tiles of %lld", (long long)bq);
  }
  // Keys the plan must cover: all of them, except that a decode-shaped causal
  // problem (16-bit, at most 64 queries) can see only its first n_q keys.
  const bool decode = dtype != MEA_F32 && nq <= 64;
  const int64_t n_keys = decode && causal && nk > nq ? nq : nk;
  CHECK(f.n_splits >= 1 && f.keys_per_split >= 1, "plan");
  CHECK((int64_t)f.n_splits * f.keys_per_split >= n_keys, "splits cover the keys (n_q %lld n_k %lld)",
        (long long)nq, (long long)nk);
  CHECK((int64_t)(f.n_splits - 1) * f.keys_per_split < n_keys, "no empty split");
  CHECK((need == 0) == (f.n_splits == 1), "workspace iff splits");
  if (f.n_splits > 1) {
    const size_t rows = (size_t)f.n_splits * (size_t)(B * H) * (size_t)nq;
    CHECK(inside(f.part_o, rows * d * 4, WS, need) && inside(f.part_m, rows * 4, WS, need) &&
              inside(f.part_l, rows * 4, WS, need),
          "partials inside the workspace (n_k %lld)", (long long)nk);
    CHECK(disjoint(f.part_o, rows * d * 4, f.part_m, rows * 4) && disjoint(f.part_m, rows * 4, f.part_l, rows * 4),
          "partials overlap");
    if (f.n_splits > mea::kCombineGroup) {
      const size_t r2 = (size_t)((f.n_splits + mea::kCombineGroup - 1) / mea::kCombineGroup) * (size_t)(B * H) * nq;
      CHECK(f.part2_o && inside(f.part2_o, r2 * d * 4, WS, need) && inside(f.part2_m, r2 * 4, WS, need) &&
                inside(f.part2_l, r2 * 4, WS, need),
            "stage buffer inside the workspace");
      CHECK(disjoint(f.part2_o, r2 * (d + 2) * 4, f.part_o, rows * (d + 2) * 4), "stage buffer overlaps");
    }
  }
}

static void check_bwd_carving(int64_t B, int64_t H, int64_t nq, int64_t d, int dtype, int out_f32, int causal = 0) {
  mea_problem p = prob(B, H, nq, 300, d, dtype, causal, 0, out_f32);
  size_t need = 0;
  CHECK(mea_attention_bwd_workspace_size(&p, &need) == MEA_OK, "bwd ws size");
  CHECK(mea_attention_bwd(&p, P, P, P, P, nullptr, P, static_cast<float*>(P), P, P, P, WS, need, nullptr) == MEA_OK,
        "bwd call");
  const mea::BwdParams& b = mea::g_last_bwd;
  const size_t rows = (size_t)(B * H) * (size_t)b.n_q_pad;
  CHECK(b.n_q_pad >= nq && b.n_q_pad % mea::kBwdRowPad == 0 && b.n_q_pad - nq < mea::kBwdRowPad, "row padding");
  // 16-bit inputs with float32 outputs keep a 16-bit copy of dO, and the
  // kernels of 16-bit outputs (and their per-row layout) then run.
  const bool do16 = dtype != MEA_F32 && out_f32;
  CHECK((b.do16 != nullptr) == do16, "dO copy carved exactly for 16-bit inputs with float32 outputs");
  // The layout the host carved is the one the kernels of this problem read.
  const bool rec = mea::bwd_two_group(dtype != MEA_F32, (int)d, (int)d, !out_f32 || do16, causal != 0, nq);
  CHECK((b.row_rec != nullptr) == rec && (b.s_init == nullptr) == rec && (b.dp_init == nullptr) == rec,
        "per-row layout matches the kernels");
  if (b.row_rec) {
    CHECK(inside(b.row_rec, rows * 16, WS, need), "records inside the workspace");
  } else {
    CHECK(inside(b.s_init, rows * 4, WS, need) && inside(b.dp_init, rows * 4, WS, need), "arrays inside");
    CHECK(disjoint(b.s_init, rows * 4, b.dp_init, rows * 4), "per-row arrays overlap");
  }
  if (b.do16) {
    const size_t cbytes = (size_t)(B * H) * (size_t)nq * (size_t)d * 2;
    CHECK(inside(b.do16, cbytes, WS, need), "dO copy inside the workspace");
    CHECK(b.row_rec ? disjoint(b.do16, cbytes, b.row_rec, rows * 16)
                    : disjoint(b.do16, cbytes, b.s_init, rows * 4) && disjoint(b.do16, cbytes, b.dp_init, rows * 4),
          "dO copy overlaps the per-row values");
  }
  CHECK(mea_attention_bwd(&p, P, P, P, P, nullptr, P, static_cast<float*>(P), P, P, P, WS, need - 1, nullptr) ==
            MEA_ERR_WORKSPACE,
        "short workspace accepted");
}

int main() {
  // Validation: every rejection happens before a launch.
  const int calls0 = mea::g_fwd_calls + mea::g_bwd_calls;
  struct Bad {
    mea_problem p;
    mea_status want;
  } bad[] = {
      {prob(1, 1, 0, 10, 64, MEA_BF16, 0), MEA_ERR_INVALID_ARG},
      {prob(1, 1, 10, 10, 96, MEA_BF16, 0), MEA_ERR_UNSUPPORTED},
      {prob(1, 1, 10, 10, 64, 9, 0), MEA_ERR_UNSUPPORTED},
      {prob(1, 1, 10, 10, 64, MEA_BF16, 3), MEA_ERR_INVALID_ARG},
      {prob(1, 1, (int64_t)1 << 31, 10, 64, MEA_BF16, 0), MEA_ERR_INVALID_ARG},
      {prob((int64_t)1 << 40, (int64_t)1 << 40, 10, 10, 64, MEA_BF16, 0), MEA_ERR_INVALID_ARG},
      {prob((int64_t)1 << 30, 4, ((int64_t)1 << 31) - 1, ((int64_t)1 << 31) - 1, 128, MEA_BF16, 0),
       MEA_ERR_INVALID_ARG},
      {prob(INT64_MAX, 1, 1, 1, 64, MEA_BF16, 0), MEA_ERR_INVALID_ARG},
      {prob(1, 1, 10, 10, 64, MEA_BF16, 0, -64), MEA_ERR_INVALID_ARG},
  };
  for (const Bad& c : bad) {
    size_t ws = 0;
    CHECK(mea_attention_fwd_workspace_size(&c.p, &ws) == c.want, "validation");
    CHECK(mea_attention_fwd(&c.p, P, P, P, P, nullptr, nullptr, WS, 1 << 30, nullptr) == c.want, "fwd validation");
    CHECK(mea_attention_bwd(&c.p, P, P, P, P, nullptr, P, static_cast<float*>(P), P, P, P, WS, 1 << 30, nullptr) ==
              c.want,
          "bwd validation");
    CHECK(mea_attention_bwd_noalloc(&c.p, P, P, P, P, nullptr, P, static_cast<float*>(P), P, P, P, nullptr) ==
              c.want,
          "noalloc validation");
  }
  // Strides near the int64 limit are rejected, not overflowed.
  mea_problem ps = prob(4, 4, 100, 100, 64, MEA_BF16, 0);
  mea_strides st;
  memset(&st, 0, sizeof(st));
  const mea_tensor_strides cont = {4 * 100 * 64, 100 * 64, 64};
  st.q = st.k = st.v = st.o = st.d_o = st.dq = st.dk = st.dv = cont;
  st.k.batch = INT64_MAX - 7;
  ps.strides = &st;
  CHECK(mea_attention_fwd(&ps, P, P, P, P, nullptr, nullptr, nullptr, 0, nullptr) == MEA_ERR_INVALID_ARG,
        "overflowing stride accepted");
  st.k = cont;
  st.dq.head = 0;
  CHECK(mea_attention_bwd(&ps, P, P, P, P, nullptr, P, static_cast<float*>(P), P, P, P, WS, 1 << 30, nullptr) ==
            MEA_ERR_INVALID_ARG,
        "output head stride 0 accepted");
  // The allocation-free backward rejects problems beyond its static scratch.
  mea_problem big = prob(1, 64, 16384 + 1, 128, 64, MEA_BF16, 0);
  CHECK(mea_attention_bwd_noalloc(&big, P, P, P, P, nullptr, P, static_cast<float*>(P), P, P, P, nullptr) ==
            MEA_ERR_SCRATCH,
        "oversized problem accepted by the allocation-free backward");
  CHECK(mea::g_fwd_calls + mea::g_bwd_calls == calls0, "a rejected call reached a launcher");
  CHECK(strlen(mea_status_string(MEA_ERR_SCRATCH)) > 10 && strcmp(mea_status_string((mea_status)77), "unknown status") == 0,
        "status strings");

  // Planning and workspace carving over a sweep of shapes.
  const int64_t nks[] = {1, 63, 64, 65, 1000, 4095, 40000, 200001, (int64_t)1 << 20, ((int64_t)1 << 22) + 3};
  for (int64_t nk : nks)
    for (int dt : {MEA_F32, MEA_BF16})
      for (int causal : {0, 1})
        for (int64_t nq : {(int64_t)1, (int64_t)100, (int64_t)300, (int64_t)4096, (int64_t)4097})
          check_fwd_plan(1, 1, nq, nk, 64, dt, causal);
  check_fwd_plan(2, 3, 256, 1 << 20, 128, MEA_F16, 0);
  // Both sides of each bound of the causal d = 64 kernel choice.
  for (int64_t nq : {(int64_t)6144, (int64_t)6145})
    check_fwd_plan(2, 64, nq, nq, 64, MEA_BF16, 1);
  for (int64_t h : {(int64_t)4, (int64_t)6}) check_fwd_plan(1, h, 32768, 32768, 64, MEA_F16, 1);
  for (int64_t nq : {(int64_t)12288, (int64_t)12800}) check_fwd_plan(1, 16, nq, nq, 64, MEA_BF16, 1);
  // Unmasked: the 4-wave kernel up to half of the two-group kernel's tile.
  for (int64_t nq : {(int64_t)256, (int64_t)257}) check_fwd_plan(2, 3, nq, 1000, 64, MEA_BF16, 0);
  for (int64_t nq : {(int64_t)128, (int64_t)129}) check_fwd_plan(2, 3, nq, 1000, 128, MEA_F16, 0);
  CHECK(mea::fwd64_bq(256, 6, false) == 128 && mea::fwd64_bq(257, 6, false) == 512 &&
            mea::fwd128_bq(128, false) == 128 && mea::fwd128_bq(129, false) == 256 && mea::fwd128_bq(100, true) == 256,
        "unmasked kernel choice");
  CHECK(mea::fwd_causal64_bq(6144, 128) == 128 && mea::fwd_causal64_bq(6145, 128) == 512 &&
            mea::fwd_causal64_bq(32768, 4) == 128 && mea::fwd_causal64_bq(32768, 6) == 512 &&
            mea::fwd_causal64_bq(12288, 16) == 128 && mea::fwd_causal64_bq(12800, 16) == 512,
        "causal d = 64 kernel choice");
  for (int64_t nq : {(int64_t)1, (int64_t)63, (int64_t)64, (int64_t)65, (int64_t)512, (int64_t)513, (int64_t)2048,
                     (int64_t)2049, (int64_t)16384})
    for (int dt : {MEA_F32, MEA_BF16})
      for (int64_t d : {(int64_t)64, (int64_t)128}) {
        for (int causal = 0; causal < 2; ++causal) {
          check_bwd_carving(2, 3, nq, d, dt, 0, causal);
          if (dt != MEA_F32) check_bwd_carving(2, 3, nq, d, dt, 1, causal);
        }
      }
  if (failures == 0) printf("abi_check ok\n");
  return failures;
}
