// Backward kernels.  The paper keeps the backward memory-efficient by
// checkpointing each chunk summary and recomputing it during
// backpropagation (Section 5.2); here the same idea is applied per tile: the
// forward saves only the per-row log-sum-exp, and every backward kernel
// recomputes the tile scores S and weights P = exp(S - lse) instead of storing
// the n_q x n_k matrix.  With D_i = dO_i . O_i the gradients are
//   dV_j = sum_i P_ij dO_i,          dP_ij = dO_i . v_j,
//   dS_ij = P_ij (dP_ij - D_i),      dQ_i = scale sum_j dS_ij k_j,
//   dK_j = scale sum_i dS_ij q_i.
// Three kernels, no atomics (bitwise reproducible):
//   pre  : D_i for every query row;
//   dkdv : one wave per 32 keys (K, V in registers), loop over query tiles;
//          lane <-> key layout, so P and dS feed the dV and dK MFMAs directly;
//   dq   : one wave per 32 queries (Q, dO in registers), loop over key tiles;
//          lane <-> query layout, so dS^T feeds the dQ^T MFMA directly.
#include "device.hpp"
#include "kernels.hpp"

// LDS fetch distances, in steps, of the two-group dQ and dK/dV kernels.
#ifndef MEA_T64_DQ_AHEAD
#define MEA_T64_DQ_AHEAD 2
#endif
#ifndef MEA_T64_DKDV_AHEAD
#define MEA_T64_DKDV_AHEAD 2
#endif
// 16-key chunks of a key tile's dS computed in the MFMA phase of the
// two-group dQ kernel (the rest in its softmax phase).
#ifndef MEA_T64_DQ_W
#define MEA_T64_DQ_W 1
#endif
// 16-query chunks of a query tile's softmax computed in the MFMA phase of the
// two-group dK/dV kernel (the rest in its softmax phase), without and with the
// causal mask.
#ifndef MEA_T64_DKDV_W
#define MEA_T64_DKDV_W 0
#endif
#ifndef MEA_T64_DKDV_WC
#define MEA_T64_DKDV_WC 1
#endif
// Keys per lane whose softmax stages the dQ kernel issues together.
#ifndef MEA_T64_DQ_G
#define MEA_T64_DQ_G 16
#endif
// K/V stages of the two-group dQ kernel's LDS ring.
#ifndef MEA_T64_DQ_NSTAGE
#define MEA_T64_DQ_NSTAGE 4
#endif

namespace mea {

template <bool B> struct BoolC { static constexpr bool value = B; };
template <int I> struct IntC { static constexpr int value = I; };

// ------------------------------------------------------------------- pre
// x as hi + mid + lo, three bf16 values (round to nearest each): the two
// differences are exact in float32, so the parts carry 24 significant bits
// and (hi + mid) + lo gives x back in float32.
__device__ __forceinline__ void split3_bf16(float x, __bf16& hi, __bf16& mid, __bf16& lo) {
  hi = (__bf16)x;
  const float r1 = x - (float)hi;
  mid = (__bf16)r1;
  lo = (__bf16)(r1 - (float)mid);
}

// D_i = dO_i . O_i and the accumulator initial values of every (padded) row,
// as records (REC) or as two float32 arrays.  For a 16-bit O with the
// forward's residual, O_i is taken as o_i + o_lo_i.  With TC != TO (float32
// o and dO, 16-bit inputs) it also writes dO rounded to TC (to nearest even,
// as the kernels' staging rounds it) to p.do16.
template <typename TO, int D, bool REC, typename TC = TO>
__global__ __launch_bounds__(256) void attn_bwd_pre_kernel(BwdParams p) {
  using T = TO;  // o and do share the output dtype
  constexpr int E = sizeof(T);
  constexpr int TPR = D * E / 16;  // threads per row, 16 bytes each
  constexpr int RPB = 256 / TPR;
  const int64_t rows = (int64_t)p.bh * p.n_q_pad;
  const int64_t prow = (int64_t)blockIdx.x * RPB + threadIdx.x / TPR;  // padded row
  const int64_t bh = prow / p.n_q_pad, i = prow % p.n_q_pad;
  const bool real = prow < rows && i < p.n_q;
  const int64_t row = bh * p.n_q + i;
  const int part = threadIdx.x % TPR;
  float acc = 0.0f;
  if (real) {
    typedef T vec16 __attribute__((ext_vector_type(16 / E)));
    const T* orow = static_cast<const T*>(p.o) + head_base(p.so, (int)bh, p.heads) + i * p.so.r;
    const T* grow = static_cast<const T*>(p.d_o) + head_base(p.sdo, (int)bh, p.heads) + i * p.sdo.r;
    // Every byte is read once: non-temporal loads (a streaming read runs about
    // 15 % faster with that cache policy).
    const vec16 o = __builtin_nontemporal_load(reinterpret_cast<const vec16*>(orow + part * (16 / E)));
    const vec16 g = __builtin_nontemporal_load(reinterpret_cast<const vec16*>(grow + part * (16 / E)));
    if constexpr (!__is_same(TC, TO)) {
      typedef TC cvec __attribute__((ext_vector_type(16 / E)));
      cvec gc;
#pragma unroll
      for (int e = 0; e < 16 / E; ++e) gc[e] = (TC)g[e];
      *reinterpret_cast<cvec*>(static_cast<TC*>(p.do16) + (bh * p.n_q + i) * D + part * (16 / E)) = gc;
    }
    float of[16 / E];
#pragma unroll
    for (int e = 0; e < 16 / E; ++e) of[e] = (float)o[e];
    if constexpr (E == 2) {
      // o + o_lo (the forward's rounding residual) is exact in float32 and
      // carries about 16 significant bits of the unrounded output.
      if (p.o_lo) {
        const vec16 lo = __builtin_nontemporal_load(reinterpret_cast<const vec16*>(
            static_cast<const T*>(p.o_lo) + (bh * p.n_q + i) * D + part * (16 / E)));
#pragma unroll
        for (int e = 0; e < 16 / E; ++e) of[e] += (float)lo[e];
      }
    }
#pragma unroll
    for (int e = 0; e < 16 / E; ++e) acc = fmaf(of[e], (float)g[e], acc);
  }
#pragma unroll
  for (int off = TPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, TPR);
  if (prow < rows && part == 0) {
    const float lse = real ? p.lse[row] : 0.0f;
    if constexpr (REC) {
      // A row with no finite lse (padding) gets weights 2^(c (S - 2^100)) = 0.
      const bool live = real && __builtin_isfinite(lse);
      const float s0 = live ? -lse / p.scale : -0x1p100f;
      const float d0 = live ? -acc : 0.0f;
      __bf16 r[8];
      split3_bf16(s0, r[0], r[1], r[2]);
      split3_bf16(d0, r[4], r[5], r[6]);
      r[3] = r[7] = (__bf16)0.0f;
      p.row_rec[prow] = __builtin_bit_cast(uint4, r);
    } else {
      // Rows with no finite lse (padding, or no visible key) get weights 0.
      const bool live = real && __builtin_isfinite(lse);
      p.s_init[prow] = live ? -lse / p.scale : -INFINITY;
      p.dp_init[prow] = live ? -acc : 0.0f;
    }
  }
}

// ------------------------------------------------------------------- dK, dV
// D: head dimension of q and k; DV: of v, o and dO.
template <typename T, int D, int DV, int QS>
struct DkdvTile {
  static constexpr int NT = 256;
  static constexpr int BKG = 128;      // keys per workgroup (32 per wave)
  static constexpr int BQ = 32 * QS;   // queries per iteration
  static constexpr int E = sizeof(T);
  static constexpr int RSQ = D + 16 / E;        // LDS row strides (elements), 16 B pad
  static constexpr int RSO = DV + 16 / E;
  static constexpr int TILEQ = BQ * RSQ;        // Q tile (elements)
  static constexpr int TILEO = BQ * RSO;        // dO tile
  static constexpr int CPRQ = D * E / 16;
  static constexpr int CPRO = DV * E / 16;
  static constexpr int CHUNKS = BQ * (CPRQ + CPRO);  // Q and dO chunks per stage
  static constexpr int CPT = (CHUNKS + NT - 1) / NT;
  static constexpr int STAGE_ELEMS = TILEQ + TILEO;
  static constexpr int STAGE_BYTES = STAGE_ELEMS * E + 2 * BQ * 4;  // + accumulator initial values
  static constexpr int LDS_BYTES = 2 * STAGE_BYTES;
  // With K_LDS the K fragments of every lane follow the two stages.
  static constexpr int KSLOT_BYTES = NT * (D / 16) * 16;
  static constexpr bool k_lds(int occ) { return E == 2 && D == 128 && occ == 2; }
  // Asynchronous stage copies (K_LDS with dO in the input dtype): each tile is
  // a whole number of 1 KiB copy units, one 16-byte slot per row chunk plus
  // one for the row pad.
  static constexpr bool async(int occ, bool same_out) { return k_lds(occ) && same_out; }
  static constexpr int UQ = (BQ * (CPRQ + 1) * 16 + 1023) / 1024;
  static constexpr int UO = (BQ * (CPRO + 1) * 16 + 1023) / 1024;
  static constexpr int ASTAGE_BYTES = (UQ + UO) * 1024 + 2 * BQ * 4;
  // SWZ (asynchronous copies with d = d_v = 128): unpadded 256-byte rows whose
  // 16-byte chunks are XOR-swizzled by the row (swz128), so that both the row
  // fragment reads and the transposing reads of Q and dO are free of bank
  // conflicts (a 16-byte row pad served the row reads only).
  static constexpr bool swz(int occ, bool same_out) { return async(occ, same_out) && D == 128 && DV == 128; }
  static constexpr int SUQ = BQ * CPRQ * 16 / 1024, SUO = BQ * CPRO * 16 / 1024;
  static constexpr int SSTAGE_BYTES = (SUQ + SUO) * 1024 + 2 * BQ * 4;
  static constexpr int stage_bytes(int occ, bool same_out) {
    return swz(occ, same_out) ? SSTAGE_BYTES : (async(occ, same_out) ? ASTAGE_BYTES : STAGE_BYTES);
  }
  static constexpr int lds_bytes(int occ, bool same_out) {
    return 2 * stage_bytes(occ, same_out) + (k_lds(occ) ? KSLOT_BYTES : 0);
  }
  static_assert(kBwdRowPad % BQ == 0, "query tiles must not pass the padded row count");
};

// Physical 16-byte chunk of logical chunk x in row r of a swizzled 256-byte
// row tile is x ^ swz128(r): a permutation of the 16 chunks over any 16
// consecutive rows (row fragment reads: 16 rows x one chunk per 16 lanes), and
// 4 consecutive rows x 4 chunks land in 4 disjoint 4-chunk groups
// (transposing reads).
__device__ __forceinline__ int swz128(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }

// Row fragment (8 elements at logical chunk x) of row r of a swizzled tile.
template <typename T>
__device__ __forceinline__ Frag<T> lds_frag_swz128(const T* tile, int r, int x) {
  return *reinterpret_cast<const Frag<T>*>(reinterpret_cast<const unsigned char*>(tile) + r * 256 +
                                           ((x ^ swz128(r)) << 4));
}

// Column fragment (as lds_col_frag) of a swizzled 256-byte row tile.
template <typename T>
__device__ __forceinline__ Frag<T> lds_col_frag_swz128(const T* tile, int row0, int col0, int lane) {
  const int g = lane >> 4, i = lane & 15;
  const int row = row0 + 8 * (g >> 1) + (i >> 2);
  const int col = col0 + 16 * (g & 1) + 4 * (i & 3);
  const unsigned char* b = reinterpret_cast<const unsigned char*>(tile);
  const int off = (col & 7) << 1;
  const v4s_t lo = lds_read_tr16(b + row * 256 + (((col >> 3) ^ swz128(row)) << 4) + off);
  const v4s_t hi = lds_read_tr16(b + (row + 4) * 256 + (((col >> 3) ^ swz128(row + 4)) << 4) + off);
  typedef short v8s_t __attribute__((ext_vector_type(8)));
  v8s_t r8;
  r8[0] = lo[0]; r8[1] = lo[1]; r8[2] = lo[2]; r8[3] = lo[3];
  r8[4] = hi[0]; r8[5] = hi[1]; r8[6] = hi[2]; r8[7] = hi[3];
  return __builtin_bit_cast(Frag<T>, r8);
}

#ifndef MEA_T128_DKDV_AHEAD
#define MEA_T128_DKDV_AHEAD 1
#endif
#ifndef MEA_DKDV_ILV
#define MEA_DKDV_ILV 1
#endif
template <typename T, typename TO, int D, int DV, int QS, int OCC, bool CAUSAL>
__global__ __launch_bounds__(256, OCC) void attn_bwd_dkdv_kernel(BwdParams p) {
  using Cfg = DkdvTile<T, D, DV, QS>;
  constexpr int RSQ = Cfg::RSQ, RSO = Cfg::RSO;
  constexpr int KC = D / 16, KCV = DV / 16;
  constexpr int NDT = D / 32, NDTV = DV / 32;
  constexpr int NQC = Cfg::BQ / 16;  // 16-query chunks per iteration

  extern __shared__ __align__(16) unsigned char smem_raw[];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int h = lane >> 5, c = lane & 31;

  const int w = xcd_remap(blockIdx.x, gridDim.x);
  const int kt_idx = w % p.n_ktiles;  // heaviest (earliest keys) first under causal
  const int bh = bh_of_group(w / p.n_ktiles, p.bh, p.heads);
  const int64_t k0 = (int64_t)kt_idx * Cfg::BKG;
  const int64_t kw = k0 + 32 * wave;
  const int64_t key = kw + c;

  const T* __restrict__ qg = static_cast<const T*>(p.q) + head_base(p.sq, bh, p.heads);
  const TO* __restrict__ dog = static_cast<const TO*>(p.d_o) + head_base(p.sdo, bh, p.heads);
  const float* __restrict__ sinitg = p.s_init + (size_t)bh * p.n_q_pad;
  const float* __restrict__ dpinitg = p.dp_init + (size_t)bh * p.n_q_pad;
  const T* __restrict__ kg = static_cast<const T*>(p.k) + head_base(p.sk, bh, p.heads);
  const T* __restrict__ vg = static_cast<const T*>(p.v) + head_base(p.sv, bh, p.heads);

  // K^T and V^T as B operands: lane (h, key c) holds row `key`, k = 16kc + 8h + s.
  // K_LDS (16-bit, d = 128, two workgroups per CU): the K fragments wait in a
  // per-lane LDS slot instead of registers (each lane reads back only what it
  // wrote, so no barrier is needed), which frees 32 registers per lane.
  constexpr bool K_LDS = Cfg::k_lds(OCC);
  // ASYNC: the Q and dO tiles go global -> LDS by asynchronous copies instead
  // of through registers (only where dO needs no conversion).
  constexpr bool ASYNC = Cfg::async(OCC, __is_same(T, TO));
  constexpr bool SWZ = Cfg::swz(OCC, __is_same(T, TO));
  constexpr int STAGE_B = Cfg::stage_bytes(OCC, __is_same(T, TO));
  constexpr int UQ = SWZ ? Cfg::SUQ : Cfg::UQ, UO = SWZ ? Cfg::SUO : Cfg::UO;  // 1 KiB copy units
  constexpr int TILEQ_L = ASYNC ? UQ * 1024 / Cfg::E : Cfg::TILEQ;  // dO tile offset (elements)
  constexpr int INIT_OFF = ASYNC ? (UQ + UO) * 1024 : Cfg::STAGE_ELEMS * Cfg::E;
  constexpr bool ILV = MEA_DKDV_ILV && sizeof(T) == 2;
  constexpr int KV_AHEAD = MEA_T128_DKDV_AHEAD;
  T* const kslot = reinterpret_cast<T*>(smem_raw + 2 * STAGE_B) + 8 * tid;
  Frag<T> kf[K_LDS ? 1 : KC], vf[KCV];
#pragma unroll
  for (int kc = 0; kc < KC; ++kc) {
    Frag<T> f;
    if (key < p.n_k) {
      f = *reinterpret_cast<const Frag<T>*>(kg + key * p.sk.r + 16 * kc + 8 * h);
    } else {
#pragma unroll
      for (int s = 0; s < 8; ++s) f[s] = (T)0.0f;
    }
    if constexpr (K_LDS) *reinterpret_cast<Frag<T>*>(kslot + 8 * Cfg::NT * kc) = f;
    else kf[kc] = f;
  }
  auto kfrag = [&](int kc) __attribute__((always_inline)) {
    if constexpr (K_LDS) return lds_frag<T>(kslot + 8 * Cfg::NT * kc);
    else return kf[kc];
  };
#pragma unroll
  for (int kc = 0; kc < KCV; ++kc) {
    if (key < p.n_k) {
      vf[kc] = *reinterpret_cast<const Frag<T>*>(vg + key * p.sv.r + 16 * kc + 8 * h);
    } else {
#pragma unroll
      for (int s = 0; s < 8; ++s) vf[kc][s] = (T)0.0f;
    }
  }

  wait_global_loads();

  f32x16 dk[NDT], dv[NDTV];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) dk[dt][r] = 0.0f;
#pragma unroll
  for (int dt = 0; dt < NDTV; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) dv[dt][r] = 0.0f;

  // Queries before the first key of this tile see none of its keys; a tile
  // past the batch's valid keys (key padding) is seen by none.
  const int64_t n_kv = valid_keys(p.kv_len, bh, p.heads, p.n_k);
  const int64_t q_begin = CAUSAL ? (k0 / Cfg::BQ) * Cfg::BQ : 0;
  const int n_iters = q_begin < p.n_q && k0 < n_kv ? (int)((p.n_q - q_begin + Cfg::BQ - 1) / Cfg::BQ) : 0;

  // Two register sets for the global -> LDS staging.  With a prefetch
  // distance PF = 2 the tile two iterations ahead is loaded into one set while
  // the other, loaded an iteration earlier, is written to LDS, so each tile's
  // loads have two iterations to land; PF = 1 (where the registers do not
  // allow two sets: float32, or two waves per SIMD) loads the next tile at the
  // start of the iteration that writes it.
  constexpr int PF = sizeof(T) == 2 && OCC == 1 ? 2 : 1;
  u32x4 stage_a[Cfg::CPT], stage_b[Cfg::CPT];
  float stage_fa = 0.0f, stage_fb = 0.0f;
  auto stage_base = [&](int buf) { return smem_raw + buf * STAGE_B; };
  auto load_stage = [&](auto set_tag, int64_t q0) __attribute__((always_inline)) {
    u32x4 (&stage)[Cfg::CPT] = decltype(set_tag)::value ? stage_b : stage_a;
    float& stage_f = decltype(set_tag)::value ? stage_fb : stage_fa;
#pragma unroll
    for (int i = 0; i < Cfg::CPT; ++i) {
      const int chunk = tid + i * Cfg::NT;
      if (chunk < Cfg::CHUNKS) {
        // The Q tile's BQ * CPRQ chunks, then the dO tile's.
        const bool is_o = chunk >= Cfg::BQ * Cfg::CPRQ;
        const int rem = is_o ? chunk - Cfg::BQ * Cfg::CPRQ : chunk;
        const int cpr = is_o ? Cfg::CPRO : Cfg::CPRQ;
        const int row = rem / cpr, col = rem % cpr;
        const int64_t q = q0 + row;
        const int64_t coff = col * (16 / Cfg::E);
        if (q >= p.n_q)
          stage[i] = u32x4{0u, 0u, 0u, 0u};
        else
          stage[i] = is_o ? ld_chunk_as<T, TO>(dog + q * p.sdo.r + coff) : ld16(qg + q * p.sq.r + coff);
      }
    }
    if (tid < 2 * Cfg::BQ) {
      // Accumulator initial value of the row (rows up to n_q_pad exist).
      const int64_t q = q0 + (tid % Cfg::BQ);
      stage_f = tid < Cfg::BQ ? sinitg[q] : dpinitg[q];
    }
  };
  auto store_stage = [&](auto set_tag, int buf) __attribute__((always_inline)) {
    const u32x4 (&stage)[Cfg::CPT] = decltype(set_tag)::value ? stage_b : stage_a;
    const float stage_f = decltype(set_tag)::value ? stage_fb : stage_fa;
    T* base = reinterpret_cast<T*>(stage_base(buf));
#pragma unroll
    for (int i = 0; i < Cfg::CPT; ++i) {
      const int chunk = tid + i * Cfg::NT;
      if (chunk < Cfg::CHUNKS) {
        const bool is_o = chunk >= Cfg::BQ * Cfg::CPRQ;
        const int rem = is_o ? chunk - Cfg::BQ * Cfg::CPRQ : chunk;
        const int cpr = is_o ? Cfg::CPRO : Cfg::CPRQ;
        const int row = rem / cpr, col = rem % cpr;
        st16(base + (is_o ? Cfg::TILEQ + row * RSO : row * RSQ) + col * (16 / Cfg::E), stage[i]);
      }
    }
    if (tid < 2 * Cfg::BQ) {
      // Initial values of the score and dP accumulators: S - lse/scale makes
      // P = 2^(c*acc) (c = scale*log2 e), dP - D makes dS = P*acc.  Rows past
      // n_q start at -inf, so their weights are 0.
      float* f = reinterpret_cast<float*>(stage_base(buf) + Cfg::STAGE_ELEMS * Cfg::E);
      f[tid] = stage_f;
    }
  };

  // ASYNC copies of a stage: unit u of the Q tile (u < UQ) or of the dO tile
  // covers slots 64 u + lane; slot s is row s / (CPR + 1), chunk s % (CPR + 1),
  // the last chunk of a row (its pad) a repeat of the one before.  Slots past
  // the tile's rows and rows past n_q copy the last valid row (finite values;
  // those queries start at -inf, so their weights are 0).  Wave w issues units
  // w, w + 4, ...; the per-row initial values go through a register as above.
  // SWZ: unit u holds rows 4u .. 4u + 3; the lane writing physical chunk
  // x = lane % 16 of row r fetches logical chunk x ^ swz128(r).
  // SWZ with a full tile (q0 + BQ <= n_q, every tile but a ragged last one):
  // wave w copies Q units w and w + 4 and dO units w and w + 4, i.e. rows
  // 4w + lane / 16 and 16 rows further, whose swizzle is the same; the per-lane
  // byte offsets are computed once and the tile's first row is a scalar base,
  // so these copies cost no vector instructions.
  constexpr bool SWZ_FAST = SWZ && UQ == 8 && UO == 8;
  const int crow = 4 * wave + (lane >> 4);
  const unsigned cch = (unsigned)(((lane & 15) ^ swz128(crow)) * 16);
  const unsigned qoff = (unsigned)(crow * p.sq.r) * Cfg::E + cch;
  const unsigned doff = (unsigned)(crow * p.sdo.r) * Cfg::E + cch;
  auto copy_stage = [&](int64_t q0, int buf) __attribute__((always_inline)) {
    if constexpr (SWZ_FAST) {
      if (q0 + Cfg::BQ <= p.n_q) {
        const T* qb = qg + q0 * p.sq.r;
        const T* db = reinterpret_cast<const T*>(dog) + q0 * p.sdo.r;
        const T* qb16 = qb + 16 * p.sq.r;
        const T* db16 = db + 16 * p.sdo.r;
        const unsigned dst =
            __builtin_amdgcn_readfirstlane(lds_addr(stage_base(buf)) + 1024u * (unsigned)wave);
        copy_to_lds16_sb(qb, qoff, dst);
        copy_to_lds16_sb(qb16, qoff, dst + 4096u);
        copy_to_lds16_sb(db, doff, dst + 8192u);
        copy_to_lds16_sb(db16, doff, dst + 12288u);
        if (tid < 2 * Cfg::BQ) {
          const int64_t q = q0 + (tid % Cfg::BQ);
          stage_fa = tid < Cfg::BQ ? sinitg[q] : dpinitg[q];
        }
        return;
      }
    }
    for (int u = __builtin_amdgcn_readfirstlane(wave); u < UQ + UO; u += 4) {
      const bool is_o = u >= UQ;
      const int uu = is_o ? u - UQ : u;
      const int cpr = is_o ? Cfg::CPRO : Cfg::CPRQ;
      int row, ch;
      if constexpr (SWZ) {
        row = 4 * uu + (lane >> 4);
        ch = (lane & 15) ^ swz128(row);
      } else {
        const int slot = 64 * uu + lane;
        row = slot / (cpr + 1);
        ch = slot % (cpr + 1);
        if (ch == cpr) ch = cpr - 1;
        if (row > Cfg::BQ - 1) row = Cfg::BQ - 1;
      }
      int64_t q = q0 + row;
      if (q > p.n_q - 1) q = p.n_q - 1;
      const T* src = (is_o ? reinterpret_cast<const T*>(dog) + q * p.sdo.r : qg + q * p.sq.r) + ch * (16 / Cfg::E);
      const unsigned dst = __builtin_amdgcn_readfirstlane(
          lds_addr(stage_base(buf) + (is_o ? UQ * 1024 : 0) + 1024 * uu));
      copy_to_lds16(src, dst);
    }
    if (tid < 2 * Cfg::BQ) {
      const int64_t q = q0 + (tid % Cfg::BQ);
      stage_fa = tid < Cfg::BQ ? sinitg[q] : dpinitg[q];
    }
  };
  // Wait for this wave's copies and loads, then write the initial values.
  auto finish_stage = [&](int buf) __attribute__((always_inline)) {
    wait_global_loads();
    if (tid < 2 * Cfg::BQ) reinterpret_cast<float*>(stage_base(buf) + INIT_OFF)[tid] = stage_fa;
  };

  const int qrow = perm32(c);
  const float cl2 = p.scale_log2;

  if constexpr (ASYNC) {
    if (n_iters > 0) {
      copy_stage(q_begin, 0);
      finish_stage(0);
    }
  } else {
    if (n_iters > 0) {
      load_stage(BoolC<false>{}, q_begin);
      store_stage(BoolC<false>{}, 0);
    }
    if (PF == 2 && n_iters > 1) load_stage(BoolC<true>{}, q_begin + Cfg::BQ);
  }
  __syncthreads();

  auto compute = [&](int it) __attribute__((always_inline)) {
    const int64_t q0 = q_begin + (int64_t)it * Cfg::BQ;
    const T* qs_t = reinterpret_cast<const T*>(stage_base(it & 1));
    const T* dos_t = qs_t + TILEQ_L;
    const float* sinit_s = reinterpret_cast<const float*>(stage_base(it & 1) + INIT_OFF);
    const float* dpinit_s = sinit_s + Cfg::BQ;

    // Nothing to do when every query of the tile precedes this wave's keys.
    const bool active = !CAUSAL || q0 + Cfg::BQ - 1 >= kw;
    if (active) {
      // Accumulators start at -lse/scale and -D of their query rows (register r
      // of lane half h holds query 32 qs + permuted_row(r, h)).
      f32x16 s[QS], dp[QS];
#pragma unroll
      for (int qs = 0; qs < QS; ++qs) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int row = 32 * qs + 16 * (j >> 1) + 8 * h + 4 * (j & 1);
          const f32x4 a = *reinterpret_cast<const f32x4*>(sinit_s + row);
          const f32x4 b = *reinterpret_cast<const f32x4*>(dpinit_s + row);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            s[qs][4 * j + e] = a[e];
            dp[qs][4 * j + e] = b[e];
          }
        }
      }
      // S = Q K^T - lse/scale and dP = dO V^T - D (rows: queries in perm32
      // order; lane: key).
      if constexpr (SWZ && QS == 1 && KV_AHEAD > 0) {
        // The Q and dO row fragments of k chunk kc are read KV_AHEAD chunks
        // before their MFMAs (a ring of registers).
        constexpr int RA = KV_AHEAD + 1;
        Frag<T> fa[RA], fg[RA];
        auto fetch = [&](int kc) __attribute__((always_inline)) {
          fa[kc % RA] = lds_frag_swz128<T>(qs_t, qrow, 2 * kc + h);
          fg[kc % RA] = lds_frag_swz128<T>(dos_t, qrow, 2 * kc + h);
        };
#pragma unroll
        for (int kc = 0; kc < KV_AHEAD; ++kc) fetch(kc);
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) {
          if (kc + KV_AHEAD < KC) fetch(kc + KV_AHEAD);
          s[0] = mma(fa[kc % RA], kfrag(kc), s[0]);
          dp[0] = mma(fg[kc % RA], vf[kc], dp[0]);
          __builtin_amdgcn_sched_barrier(0);
        }
      } else
#pragma unroll
      for (int kc = 0; kc < (KC > KCV ? KC : KCV); ++kc) {
#pragma unroll
        for (int qs = 0; qs < QS; ++qs) {
          if (kc < KC) {
            const Frag<T> a = SWZ ? lds_frag_swz128<T>(qs_t, 32 * qs + qrow, 2 * kc + h)
                                  : lds_frag<T>(qs_t + (32 * qs + qrow) * RSQ + 16 * kc + 8 * h);
            s[qs] = mma(a, kfrag(kc), s[qs]);
          }
          if (kc < KCV) {
            const Frag<T> g = SWZ ? lds_frag_swz128<T>(dos_t, 32 * qs + qrow, 2 * kc + h)
                                  : lds_frag<T>(dos_t + (32 * qs + qrow) * RSO + 16 * kc + 8 * h);
            dp[qs] = mma(g, vf[kc], dp[qs]);
          }
        }
      }
      const bool need_mask = CAUSAL && q0 < kw + 31;
      // The mask applies to the tiles on the diagonal only: a uniform branch
      // keeps its compares out of the other tiles (the empty volatile
      // statement keeps the compiler from turning it into selects).  A masked
      // score becomes -inf, so its weight 2^(c S) is exactly 0.
      if (need_mask) {
        asm volatile("");
#pragma unroll
        for (int qs = 0; qs < QS; ++qs) {
          const int key_rel = (int)(key - q0);  // key minus the tile's first query
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (key_rel > 32 * qs + permuted_row(r, h)) s[qs][r] = -INFINITY;
        }
      }
      auto col_o = [&](int qc, int dt) __attribute__((always_inline)) {
        if constexpr (SWZ) return lds_col_frag_swz128<T>(dos_t, 16 * qc, 32 * dt, lane);
        else if constexpr (sizeof(T) == 2) return lds_col_frag<T>(dos_t, RSO, 16 * qc, 32 * dt, lane);
        else return lds_col_frag_f32(reinterpret_cast<const float*>(dos_t), RSO, 16 * qc, 32 * dt, lane);
      };
      auto col_q = [&](int qc, int dt) __attribute__((always_inline)) {
        if constexpr (SWZ) return lds_col_frag_swz128<T>(qs_t, 16 * qc, 32 * dt, lane);
        else if constexpr (sizeof(T) == 2) return lds_col_frag<T>(qs_t, RSQ, 16 * qc, 32 * dt, lane);
        else return lds_col_frag_f32(reinterpret_cast<const float*>(qs_t), RSQ, 16 * qc, 32 * dt, lane);
      };
      constexpr int NDTM = NDT > NDTV ? NDT : NDTV;
      if constexpr (ILV) {
        // The weights of 16-query chunk qc + 1 (P = 2^(c S), dS = P (dP - D),
        // rounded to fragments) are computed between the dV/dK MFMAs of chunk
        // qc, a share per step, so this wave's VALU work overlaps its own
        // MFMAs; each step's LDS operands are read one step ahead.
        static_assert(8 % (2 * NDTM) == 0, "score pairs per step");
        constexpr int PER = 8 / NDTM;
        typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
        u32x4v pw, dw;  // chunk qc + 1 as bf16 pairs
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          const float p0 = fast_exp2(s[0][e] * cl2), p1 = fast_exp2(s[0][e + 1] * cl2);
          pw[e / 2] = pack2<T>(p0, p1);
          dw[e / 2] = pack2<T>(p0 * dp[0][e], p1 * dp[0][e + 1]);
        }
        Frag<T> pa = __builtin_bit_cast(Frag<T>, pw), da = __builtin_bit_cast(Frag<T>, dw);
        Frag<T> bo = col_o(0, 0), bq = col_q(0, 0);
#pragma unroll
        for (int qc = 0; qc < NQC; ++qc) {
#pragma unroll
          for (int dt = 0; dt < NDTM; ++dt) {
            const bool last = dt + 1 == NDTM;
            const int nqc = last ? qc + 1 : qc, ndt = last ? 0 : dt + 1;
            Frag<T> bo_n = bo, bq_n = bq;
            if (nqc < NQC) {
              if (ndt < NDTV) bo_n = col_o(nqc, ndt);
              if (ndt < NDT) bq_n = col_q(nqc, ndt);
            }
            if (dt < NDTV) dv[dt] = mma(pa, bo, dv[dt]);
            if (dt < NDT) dk[dt] = mma(da, bq, dk[dt]);
            if (qc + 1 < NQC) {
              const f32x16& sn = s[(qc + 1) >> 1];
              const f32x16& dn = dp[(qc + 1) >> 1];
#pragma unroll
              for (int e = PER * dt; e < PER * dt + PER; e += 2) {
                const int r = 8 * ((qc + 1) & 1) + e;
                const float p0 = fast_exp2(sn[r] * cl2), p1 = fast_exp2(sn[r + 1] * cl2);
                pw[e / 2] = pack2<T>(p0, p1);
                dw[e / 2] = pack2<T>(p0 * dn[r], p1 * dn[r + 1]);
              }
            }
            bo = bo_n;
            bq = bq_n;
            __builtin_amdgcn_sched_barrier(0);
          }
          if (qc + 1 < NQC) {
            pa = __builtin_bit_cast(Frag<T>, pw);
            da = __builtin_bit_cast(Frag<T>, dw);
          }
        }
      } else {
#pragma unroll
        for (int qs = 0; qs < QS; ++qs) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float pr = fast_exp2(s[qs][r] * cl2);
            s[qs][r] = pr;                // P
            dp[qs][r] = pr * dp[qs][r];   // dS = P (dP - D)
          }
        }
        // dV += P^T dO and dK += dS^T Q (A: lane = key row, k = queries).
#pragma unroll
        for (int qc = 0; qc < NQC; ++qc) {
          float tp[8], td[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            tp[e] = s[qc >> 1][8 * (qc & 1) + e];
            td[e] = dp[qc >> 1][8 * (qc & 1) + e];
          }
          const Frag<T> pa = to_frag<T>(tp);
          const Frag<T> da = to_frag<T>(td);
#pragma unroll
          for (int dt = 0; dt < NDTM; ++dt) {
            if (dt < NDTV) dv[dt] = mma(pa, col_o(qc, dt), dv[dt]);
            if (dt < NDT) dk[dt] = mma(da, col_q(qc, dt), dk[dt]);
          }
        }
      }
    }
  };
  // Iteration it computes tile it from LDS buffer it & 1 and writes tile
  // it + 1 to the other LDS buffer.  PF = 2: set A holds even tiles, set B
  // odd ones, and tile it + 2 is loaded into the set that held tile it;
  // PF = 1: tile it + 1 is loaded into set A in this iteration.
  if constexpr (PF == 2) {
    auto step = [&](auto odd_tag, int it) __attribute__((always_inline)) {
      constexpr bool ODD = decltype(odd_tag)::value;
      if (it + 2 < n_iters) load_stage(BoolC<ODD>{}, q_begin + (int64_t)(it + 2) * Cfg::BQ);
      compute(it);
      if (it + 1 < n_iters) store_stage(BoolC<!ODD>{}, (it + 1) & 1);
      __syncthreads();
    };
    for (int it = 0; it < n_iters; it += 2) {
      step(BoolC<false>{}, it);
      if (it + 1 < n_iters) step(BoolC<true>{}, it + 1);
    }
  } else {
    for (int it = 0; it < n_iters; ++it) {
      const bool has_next = it + 1 < n_iters;
      if constexpr (ASYNC) {
        if (has_next) copy_stage(q_begin + (int64_t)(it + 1) * Cfg::BQ, (it + 1) & 1);
        compute(it);
        if (has_next) finish_stage((it + 1) & 1);
      } else {
        if (has_next) load_stage(BoolC<false>{}, q_begin + (int64_t)(it + 1) * Cfg::BQ);
        compute(it);
        if (has_next) store_stage(BoolC<false>{}, (it + 1) & 1);
      }
      __syncthreads();
    }
  }

  // Accumulators: lane (h, feature c), register r <-> key kw + c_row(r, h).
  T* dkg = static_cast<T*>(p.dk) + head_base(p.sdk, bh, p.heads);
  T* dvg = static_cast<T*>(p.dv) + head_base(p.sdv, bh, p.heads);
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t kr = kw + c_row(r, h);
      if (kr < p.n_k)  // keys past the valid length get zero gradients
        dkg[kr * p.sdk.r + 32 * dt + c] = kr < n_kv ? (T)(dk[dt][r] * p.scale) : (T)0.0f;
    }
#pragma unroll
  for (int dt = 0; dt < NDTV; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t kr = kw + c_row(r, h);
      if (kr < p.n_k) dvg[kr * p.sdv.r + 32 * dt + c] = kr < n_kv ? (T)dv[dt][r] : (T)0.0f;
    }
}

// -------------------------------------------------- dK, dV (two groups)
// 16-bit inputs and outputs, d = 64.  Eight waves of 32 keys each (K and V in
// registers, dK and dV accumulated in registers) in two groups of four that
// alternate an MFMA phase and a VALU phase, separated by workgroup barriers;
// group 1 runs one phase behind group 0, so waves w and w + 4, which share a
// SIMD, always have different roles.  MFMA phase of query tile i: dV += P^T dO
// and dK += dS^T Q for tile i - 1, then S = Q K^T and dP = dO V^T for tile i.
// VALU phase of tile i: P = 2^(c S), dS = P dP (the accumulators start at
// -lse/scale and -D), rounded into the operands of the next MFMA phase.
// Q, dO and the initial values stream through a four-stage LDS ring with
// asynchronous global -> LDS copies issued by group 1.
namespace kvpp {
constexpr int D = 64, NW = 8, BKG = NW * 32, BQ = 64, QS = BQ / 32, NSTAGE = 4;
constexpr int RSB = 144;                      // bytes per LDS row (128 + 16 pad)
constexpr int TILEB = BQ * RSB;               // one Q or dO tile: 9 KiB
constexpr int RECB = BQ * 16;                 // the tile's per-row records
constexpr int STAGEB = 2 * TILEB + RECB;      // 19456 bytes
constexpr int UNITS = 2 * TILEB / 1024 + 1;   // 1 KiB copies per stage (18 + 1)
static_assert(TILEB % 1024 == 0 && RECB == 1024, "stage layout");
}  // namespace kvpp

// MFMA-phase step order of the two-group dK/dV kernel when part of the
// softmax moves into that phase (steps of two MFMAs): 0, 1 dV/dK of query
// chunk 0 of the previous tile (dt = 0, 1); 2..5 S/dP of query sub-tile 0 of
// this tile (kc = 0..3); 6..11 dV/dK of chunks 1..3; 12..15 S/dP of sub-tile 1.
struct KvStep {
  int dvdk;  // 1: dV/dK step (a = query chunk, b = dt); 0: S/dP (a = qs, b = kc)
  int a, b;
};
__device__ constexpr KvStep kv_step_split(int g) {
  return g < 2 ? KvStep{1, 0, g}
       : g < 6 ? KvStep{0, 0, g - 2}
       : g < 12 ? KvStep{1, 1 + (g - 6) / 2, (g - 6) % 2}
                : KvStep{0, 1, g - 12};
}

template <typename T, bool CAUSAL>
__global__ __launch_bounds__(512, 1) void attn_bwd_dkdv_pp_kernel(BwdParams p) {
  using namespace kvpp;
  static_assert(sizeof(T) == 2, "16-bit inputs only");
  constexpr int KC = D / 16, NDT = D / 32, NQC = BQ / 16;
  __shared__ __align__(16) unsigned char smem[NSTAGE * STAGEB];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2;
  const int lane = tid & 63;
  const int h = lane >> 5, c = lane & 31;

  const int w = xcd_remap(blockIdx.x, gridDim.x);
  const int kt_idx = w % p.n_ktiles;
  const int bh = bh_of_group(w / p.n_ktiles, p.bh, p.heads);
  const int64_t k0 = (int64_t)kt_idx * BKG;
  const int64_t kw = k0 + 32 * wave;
  const int64_t key = kw + c;

  const T* __restrict__ qg = static_cast<const T*>(p.q) + head_base(p.sq, bh, p.heads);
  const T* __restrict__ dog = static_cast<const T*>(p.d_o) + head_base(p.sdo, bh, p.heads);
  const uint4* __restrict__ recg = p.row_rec + (size_t)bh * p.n_q_pad;
  const T* __restrict__ kg = static_cast<const T*>(p.k) + head_base(p.sk, bh, p.heads);
  const T* __restrict__ vg = static_cast<const T*>(p.v) + head_base(p.sv, bh, p.heads);

  Frag<T> kf[KC], vf[KC];
#pragma unroll
  for (int kc = 0; kc < KC; ++kc) {
    if (key < p.n_k) {
      kf[kc] = *reinterpret_cast<const Frag<T>*>(kg + key * p.sk.r + 16 * kc + 8 * h);
      vf[kc] = *reinterpret_cast<const Frag<T>*>(vg + key * p.sv.r + 16 * kc + 8 * h);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        kf[kc][e] = (T)0.0f;
        vf[kc][e] = (T)0.0f;
      }
    }
  }
  wait_global_loads();

  f32x16 dk[NDT], dv[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      dk[dt][r] = 0.0f;
      dv[dt][r] = 0.0f;
    }

  // Queries before the workgroup's first key see none of its keys (causal);
  // a workgroup past the batch's valid keys (key padding) is seen by none.
  const int64_t n_kv = valid_keys(p.kv_len, bh, p.heads, p.n_k);
  const int64_t q_begin = CAUSAL ? (k0 / BQ) * BQ : 0;
  const int n_iters = q_begin < p.n_q && k0 < n_kv ? (int)((p.n_q - q_begin + BQ - 1) / BQ) : 0;
  auto stage = [&](int i) { return smem + (i % NSTAGE) * STAGEB; };

  // Copy unit u (0 <= u < UNITS) of query tile i into its stage: units 0..8
  // are the Q tile, 9..17 the dO tile (lane slot s = 64 (u % 9) + lane is row
  // s / 9, 16-byte chunk s % 9; chunk 8 is the row pad and gets a copy of
  // chunk 7), unit 18 the per-row records (lane l: row l; the padded record
  // array holds every row of the tile).  Query rows past n_q repeat the last
  // row (finite values; their weights are 0).
  const int n_full = n_iters > 0 ? (int)((p.n_q - q_begin) / BQ) : 0;  // tiles with no row past n_q
  auto unit_row = [&](int u) { return (64 * (u % 9) + lane) / 9; };
  auto unit_col = [&](int u) {
    const int ch = (64 * (u % 9) + lane) % 9;
    return (unsigned)(16 * (ch < 8 ? ch : 7));
  };
  // Byte offset within a tile (row strides < 2^24 elements, checked on the host).
  auto unit_off = [&](int u) {
    const unsigned rsb = (unsigned)sizeof(T) * (unsigned)(u >= 9 ? p.sdo.r : p.sq.r);
    return (unsigned)unit_row(u) * rsb + unit_col(u);
  };
  auto copy_unit = [&](int i, int u, unsigned off) __attribute__((always_inline)) {
    const int64_t q0 = q_begin + (int64_t)i * BQ;
    unsigned char* st = stage(i);
    if (u < UNITS - 1) {
      const int which = u >= 9, v9 = u - 9 * which;
      const T* g = which ? dog : qg;
      const int64_t rs = which ? p.sdo.r : p.sq.r;
      const unsigned lds = __builtin_amdgcn_readfirstlane(lds_addr(st + which * TILEB + 1024 * v9));
      if (i < n_full) {
        copy_to_lds16_sb(g + q0 * rs, off, lds);
      } else {
        int64_t q = q0 + unit_row(u);
        if (q > p.n_q - 1) q = p.n_q - 1;
        copy_to_lds16(reinterpret_cast<const unsigned char*>(g + q * rs) + unit_col(u), lds);
      }
    } else {
      copy_to_lds16(recg + q0 + lane, __builtin_amdgcn_readfirstlane(lds_addr(st + 2 * TILEB)));
    }
  };
  // Each wave's share of the copies of a tile: units wave + 8k (three for
  // waves 0..2, two for the others), with the lane's byte offset within the
  // tile of each unit computed once (a tile that ends past n_q takes the
  // clamped path).
  constexpr int MAXU = (UNITS + NW - 1) / NW;
  const int n_units = (UNITS - wave + NW - 1) / NW;
  unsigned uoff[MAXU];
#pragma unroll
  for (int k = 0; k < MAXU; ++k) {
    const int u = wave + NW * k;
    uoff[k] = u < UNITS - 1 ? unit_off(u) : 0u;
  }
  auto issue = [&](int i) __attribute__((always_inline)) {
    if (i < n_iters) {
#pragma unroll
      for (int k = 0; k < MAXU; ++k)
        if (wave + NW * k < UNITS) copy_unit(i, wave + NW * k, uoff[k]);
    }
  };
  // Wait until this wave's copies of older tiles have landed; those of the
  // tile issued last (`recent` says whether it exists) may still run.
  auto wait_copies = [&](bool recent) __attribute__((always_inline)) {
    if (!recent) wait_global_loads();
    else if (n_units == 3) wait_global_loads_upto<3>();
    else wait_global_loads_upto<2>();
  };
  auto barrier = [&]() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" ::: "memory");
  };

  // Copy schedule: group 1 issues its share of tile j in its VALU phase of
  // tile j - 3, group 0 in its VALU phase of tile j - 2; each group waits for
  // its share before the barrier that precedes group 0's first read of tile j
  // (the end of group 1's MFMA phase, and of group 0's VALU phase, of tile
  // j - 1).  A stage is overwritten only after group 1's MFMA phase of the
  // tile four earlier, its last reader, has ended.
  // Prologue: all waves copy tile 0; group 1 then issues its shares of tiles
  // 1 and 2, group 0 its share of tile 1, and group 1 starts one phase behind.
  if (n_iters > 0)
    for (int u = wave; u < UNITS; u += NW) copy_unit(0, u, u < UNITS - 1 ? unit_off(u) : 0u);
  wait_global_loads();
  __syncthreads();
  if (grp == 1) {
    issue(1);
    issue(2);
    barrier();
  } else {
    issue(1);
  }

  const int qrow = perm32(c);
  const float cl2 = p.scale_log2;
  f32x16 s[QS], dp[QS];
  Frag<T> pa[NQC], da[NQC];
  // The MFMA phase issues each LDS fragment read AHEAD steps (two MFMAs each)
  // before its MFMAs (scheduling fences between steps), so that a wave alone
  // on the matrix pipe does not wait for LDS latency.  The causal variant keeps
  // a shorter distance for its larger register footprint.
  constexpr int AHEAD = CAUSAL ? 2 : MEA_T64_DKDV_AHEAD;
  // One fetch ring serves the whole MFMA phase.  Steps 0 .. NS1 - 1 are
  // dV += P^T dO and dK += dS^T Q of the previous tile (column fragments of dO
  // and Q: k = queries); steps NS1 .. NS1 + NS2 - 1 are S = Q K^T + s_init and
  // dP = dO V^T + dp_init of this tile (row fragments of Q and dO).  A step's
  // two fragments are read AHEAD steps before its MFMAs: across the move from
  // dV/dK to S/dP, and, for the first AHEAD steps, at the end of the preceding
  // softmax phase, so that the phase never starts on LDS latency.
  constexpr int NS1 = NQC * NDT, NS2 = KC * QS, NS = NS1 + NS2;
  Frag<T> rx[AHEAD + 1], ry[AHEAD + 1];
  auto fetch = [&](int i_dv, int i_sd, int g) __attribute__((always_inline)) {
    const int slot = g % (AHEAD + 1);
    if (g < NS1) {
      const unsigned char* st = stage(i_dv);
      const int qc = g / NDT, dt = g % NDT;
      rx[slot] = lds_col_frag<T>(reinterpret_cast<const T*>(st + TILEB), RSB / 2, 16 * qc, 32 * dt, lane);
      ry[slot] = lds_col_frag<T>(reinterpret_cast<const T*>(st), RSB / 2, 16 * qc, 32 * dt, lane);
    } else {
      const unsigned char* st = stage(i_sd);
      const int kc = (g - NS1) / QS, qs = (g - NS1) % QS;
      const int off = (32 * qs + qrow) * (RSB / 2) + 16 * kc + 8 * h;
      rx[slot] = lds_frag<T>(reinterpret_cast<const T*>(st) + off);
      ry[slot] = lds_frag<T>(reinterpret_cast<const T*>(st + TILEB) + off);
    }
  };
  // S and dP start from the per-row values of tile i: one bf16 MFMA each per
  // query sub-tile, A = the rows' records (lane c: query 32 qs + perm32(c),
  // the same record in both lane halves), B = ones picking the three s parts
  // (bsel_s) or the three d parts (bsel_d) in the first lane half and zeros in
  // the second, C = 0.  The records are read at the start of the MFMA phase.
  bf16x8 rec[QS];
  bf16x8 bsel_s, bsel_d;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    bsel_s[e] = (__bf16)(h == 0 && e < 3 ? 1.0f : 0.0f);
    bsel_d[e] = (__bf16)(h == 0 && e >= 4 && e < 7 ? 1.0f : 0.0f);
  }
  auto read_rec = [&](int i) __attribute__((always_inline)) {
#pragma unroll
    for (int qs = 0; qs < QS; ++qs)
      rec[qs] = *reinterpret_cast<const bf16x8*>(stage(i) + 2 * TILEB + 16 * (32 * qs + qrow));
  };
  auto init_sdp_qs = [&](int qs) __attribute__((always_inline)) {
    const f32x16 zero = {};
    s[qs] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(rec[qs], bsel_s, zero, 0, 0, 0);
    dp[qs] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(rec[qs], bsel_d, zero, 0, 0, 0);
  };
  auto init_sdp = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) init_sdp_qs(qs);
  };
  // Steps [G0, G1) with dV/dK of tile i_dv and S/dP of tile i_sd; the ring
  // already holds steps G0 .. G0 + AHEAD - 1.  S and dP are initialised just
  // before their first step.
  auto run = [&](auto g0_tag, auto g1_tag, int i_dv, int i_sd) __attribute__((always_inline)) {
    constexpr int G0 = decltype(g0_tag)::value, G1 = decltype(g1_tag)::value;
#pragma unroll
    for (int g = G0; g < G1; ++g) {
      if (g + AHEAD < G1) fetch(i_dv, i_sd, g + AHEAD);
      if (g == NS1) init_sdp();
      const int slot = g % (AHEAD + 1);
      if (g < NS1) {
        const int qc = g / NDT, dt = g % NDT;
        dv[dt] = mma(pa[qc], rx[slot], dv[dt]);
        dk[dt] = mma(da[qc], ry[slot], dk[dt]);
      } else {
        const int kc = (g - NS1) / QS, qs = (g - NS1) % QS;
        s[qs] = mma(rx[slot], kf[kc], s[qs]);
        dp[qs] = mma(ry[slot], vf[kc], dp[qs]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // dV/dK of tile i_dv alone (the ring was filled at the end of the softmax
  // phase of tile i_dv).
  auto dvdk = [&](int i_dv) __attribute__((always_inline)) { run(IntC<0>{}, IntC<NS1>{}, i_dv, i_dv); };

  // Softmax of the first W 16-query chunks of a tile in its MFMA phase (the
  // steady-state MFMA phase then takes the step order of kv_step_split).  In
  // that order S and dP of sub-tile 0 are final after step 5, and chunk c is
  // written only after the dV/dK step that reads the old chunk c (steps 1 and
  // 7); half-chunk u (four queries per lane) is issued in step 7 + 4u / W,
  // after the step's two MFMAs, and runs while they execute.  The first two
  // steps are the same in both orders, so the softmax phase's ring prefetch
  // serves either.
  constexpr int W = CAUSAL ? MEA_T64_DKDV_WC : MEA_T64_DKDV_W;
  static_assert(W >= 0 && W <= 2, "only chunks of query sub-tile 0 are final before the dV/dK steps");
  static_assert(W == 0 || AHEAD <= 2, "the prefetched steps must be dV/dK steps of chunk 0");
  static_assert(NS1 == 8 && NS2 == 8 && QS == 2 && NDT == 2 && KC == 4, "step table shape");
  // P = 2^(c S) and dS = P dP for four queries of chunk c (half hf), masked
  // like the softmax phase, rounded and packed two per dword.
  auto pd_half = [&](int cidx, int hf, bool need_mask, int key_rel, u32x2& pw, u32x2& dw)
      __attribute__((always_inline)) {
    const int qs = cidx >> 1;
    float pr[4], ds[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = 8 * (cidx & 1) + 4 * hf + e;
      float x = fast_exp2(s[qs][r] * cl2);
      if (need_mask && key_rel > 32 * qs + permuted_row(r, h)) x = 0.0f;
      pr[e] = x;
      ds[e] = x * dp[qs][r];
    }
    pw = u32x2{pack2<T>(pr[0], pr[1]), pack2<T>(pr[2], pr[3])};
    dw = u32x2{pack2<T>(ds[0], ds[1]), pack2<T>(ds[2], ds[3])};
  };
  auto run_split = [&](int i_dv, int i_sd, bool need_mask, int key_rel) __attribute__((always_inline)) {
    constexpr int NSS = NS1 + NS2;
    auto fetch_split = [&](int g) __attribute__((always_inline)) {
      const int slot = g % (AHEAD + 1);
      const KvStep k = kv_step_split(g);
      if (k.dvdk) {
        const unsigned char* st = stage(i_dv);
        rx[slot] = lds_col_frag<T>(reinterpret_cast<const T*>(st + TILEB), RSB / 2, 16 * k.a, 32 * k.b, lane);
        ry[slot] = lds_col_frag<T>(reinterpret_cast<const T*>(st), RSB / 2, 16 * k.a, 32 * k.b, lane);
      } else {
        const unsigned char* st = stage(i_sd);
        const int off = (32 * k.a + qrow) * (RSB / 2) + 16 * k.b + 8 * h;
        rx[slot] = lds_frag<T>(reinterpret_cast<const T*>(st) + off);
        ry[slot] = lds_frag<T>(reinterpret_cast<const T*>(st + TILEB) + off);
      }
    };
    u32x2 pw0 = {0u, 0u}, dw0 = {0u, 0u};
#pragma unroll
    for (int g = 0; g < NSS; ++g) {
      if (g + AHEAD < NSS) fetch_split(g + AHEAD);
      if (g == 2) init_sdp_qs(0);
      if (g == 12) init_sdp_qs(1);
      const int slot = g % (AHEAD + 1);
      const KvStep k = kv_step_split(g);
      if (k.dvdk) dv[k.b] = mma(pa[k.a], rx[slot], dv[k.b]);
      else s[k.a] = mma(rx[slot], kf[k.b], s[k.a]);
      int u = -1;
      if constexpr (W > 0) {
#pragma unroll
        for (int uu = 0; uu < 2 * W; ++uu)
          if (g == 7 + (4 * uu) / W) u = uu;
      }
      if (k.dvdk) dk[k.b] = mma(da[k.a], ry[slot], dk[k.b]);
      else dp[k.a] = mma(ry[slot], vf[k.b], dp[k.a]);
      if (u >= 0) {
        u32x2 pw, dw;
        pd_half(u >> 1, u & 1, need_mask, key_rel, pw, dw);
        if ((u & 1) == 0) {
          pw0 = pw;
          dw0 = dw;
        } else {
          pa[u >> 1] = __builtin_bit_cast(Frag<T>, u32x4{pw0[0], pw0[1], pw[0], pw[1]});
          da[u >> 1] = __builtin_bit_cast(Frag<T>, u32x4{dw0[0], dw0[1], dw[0], dw[1]});
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // One iteration per query tile.  MODE 0: the tile is not active for this
  // wave (causal: all its queries precede the wave's keys), only the copies
  // and barriers run; MODE 1: the wave's first active tile (S/dP only); MODE 2:
  // dV/dK of the previous tile and S/dP of this one.  A tile active for a wave
  // stays active for its later tiles (the queries only grow), so the modes
  // come in this order and each loop below runs one of them.
  auto iteration = [&](auto mode_tag, auto mask_tag, int i) __attribute__((always_inline)) {
    constexpr int MODE = decltype(mode_tag)::value;
    const int64_t q0 = q_begin + (int64_t)i * BQ;
    // MASK: the tile may hold queries before some of the wave's keys; the
    // tiles after those are compiled without the compare and select per score.
    const bool need_mask = decltype(mask_tag)::value && q0 < kw + 31;
    const int key_rel = (int)(key - q0);  // key minus the tile's first query
    // ---- MFMA phase (S and dP are free: the last softmax phase converted them)
    mfma_phase_priority();
    if constexpr (MODE == 1) {
      read_rec(i);
#pragma unroll
      for (int g = NS1; g < NS1 + AHEAD; ++g) fetch(i, i, g);
      run(IntC<NS1>{}, IntC<NS>{}, i, i);
    } else if constexpr (MODE == 2) {
      read_rec(i);
      if constexpr (W > 0) run_split(i - 1, i, need_mask, key_rel);
      else run(IntC<0>{}, IntC<NS>{}, i - 1, i);
    }
    // Group 1: tile i + 1 must land before this barrier (its share of tile
    // i + 2 may still run).
    if (grp == 1) wait_copies(i + 2 < n_iters);
    barrier();
    // ---- VALU phase
    valu_phase_priority();
    if constexpr (MODE != 0) {
      // Chunks C0 .. NQC - 1 (the MFMA phase of a steady-state tile did the
      // first W).
      constexpr int C0 = MODE == 2 ? W : 0;
#pragma unroll
      for (int qs = 0; qs < QS; ++qs)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          if (2 * qs + r / 8 < C0) continue;
          float pr = fast_exp2(s[qs][r] * cl2);
          if (need_mask && key_rel > 32 * qs + permuted_row(r, h)) pr = 0.0f;
          s[qs][r] = pr;
          dp[qs][r] = pr * dp[qs][r];
        }
#pragma unroll
      for (int qc = C0; qc < NQC; ++qc) {
        float tp[8], td[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          tp[e] = s[qc >> 1][8 * (qc & 1) + e];
          td[e] = dp[qc >> 1][8 * (qc & 1) + e];
        }
        pa[qc] = to_frag<T>(tp);
        da[qc] = to_frag<T>(td);
        keep_here(pa[qc]);  // the conversions belong to this phase
        keep_here(da[qc]);
      }
      // The first fragments of dV/dK of this tile, for the next MFMA phase.
#pragma unroll
      for (int g = 0; g < AHEAD; ++g) fetch(i, i, g);
    }
    if (grp == 1) {
      issue(i + 3);
    } else {
      // Group 0: its share of tile i + 2, then wait for tile i + 1.
      issue(i + 2);
      wait_copies(i + 2 < n_iters);
    }
    barrier();
  };
  // The wave's first active tile: the first i with q_begin + 64 i + 63 >= kw.
  int i_first = 0;
  if (CAUSAL) {
    const int64_t t = kw - q_begin - (BQ - 1);
    i_first = t > 0 ? (int)((t + BQ - 1) / BQ) : 0;
    if (i_first > n_iters) i_first = n_iters;
  }
  // Tiles from i_plain on start at or after query kw + 31: no query of theirs
  // precedes a key of the wave, so they need no mask.
  int i_plain = 0;
  if (CAUSAL) {
    const int64_t t = kw + 31 - q_begin;
    i_plain = t > 0 ? (int)((t + BQ - 1) / BQ) : 0;
    if (i_plain > n_iters) i_plain = n_iters;
  }
  int i = 0;
  for (; i < i_first; ++i) iteration(IntC<0>{}, BoolC<false>{}, i);
  if (i < n_iters) iteration(IntC<1>{}, BoolC<CAUSAL>{}, i++);
  for (; i < i_plain; ++i) iteration(IntC<2>{}, BoolC<CAUSAL>{}, i);
  for (; i < n_iters; ++i) iteration(IntC<2>{}, BoolC<false>{}, i);
  // dV/dK of the last tile.
  if (i_first < n_iters) dvdk(n_iters - 1);
  // Group 0 issued one barrier fewer (group 1's start delay): balance it so
  // that no wave leaves while the other group still waits at a barrier.
  if (grp == 0) barrier();

  T* dkg = static_cast<T*>(p.dk) + head_base(p.sdk, bh, p.heads);
  T* dvg = static_cast<T*>(p.dv) + head_base(p.sdv, bh, p.heads);
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t kr = kw + c_row(r, h);
      if (kr < p.n_k) {  // keys past the valid length get zero gradients
        dkg[kr * p.sdk.r + 32 * dt + c] = kr < n_kv ? (T)(dk[dt][r] * p.scale) : (T)0.0f;
        dvg[kr * p.sdv.r + 32 * dt + c] = kr < n_kv ? (T)dv[dt][r] : (T)0.0f;
      }
    }
}

// ------------------------------------------------------------------- dQ
// D: head dimension of q and k; DV: of v and dO.
#ifndef MEA_T128_DQ_AHEAD
#define MEA_T128_DQ_AHEAD 1
#endif
#ifndef MEA_T128_DQ_SWZ
#define MEA_T128_DQ_SWZ 1
#endif
template <typename T, typename TO, int D, int DV, int QT, int BK, int OCC, bool CAUSAL>
__global__ __launch_bounds__(256, OCC) void attn_bwd_dq_kernel(BwdParams p) {
  constexpr int NT = 256;
  constexpr int BQ = 128 * QT;  // 4 waves x QT x 32 queries
  constexpr int E = sizeof(T);
  constexpr int RSK = D + 16 / E, RSV = DV + 16 / E;  // LDS row strides (elements), 16 B pad
  constexpr int TILEK = BK * RSK, TILEV = BK * RSV;
  constexpr int CPRK = D * E / 16, CPRV = DV * E / 16;
  constexpr int CHUNKS = BK * (CPRK + CPRV);
  constexpr int CPT = CHUNKS / NT;
  static_assert(CHUNKS % NT == 0, "tile must split evenly");
  constexpr int KC = D / 16, KCV = DV / 16;
  constexpr int NKT = BK / 32;
  constexpr int NPC = BK / 16;
  constexpr int NDT = D / 32;
  // SWZ (16-bit, d = d_v = 128, 32-key tiles): the K and V tiles go global ->
  // LDS by asynchronous copies into unpadded 256-byte rows whose 16-byte
  // chunks are XOR-swizzled by the row (swz128), which keeps the row and the
  // transposing reads free of bank conflicts and frees the staging registers.
  constexpr bool SWZ = MEA_T128_DQ_SWZ && sizeof(T) == 2 && D == 128 && DV == 128 && BK == 32;
  constexpr int TK = SWZ ? BK * D : TILEK, TV = SWZ ? BK * DV : TILEV;  // tile sizes (elements)
  constexpr int DQ_AHEAD = MEA_T128_DQ_AHEAD;

  extern __shared__ __align__(16) unsigned char smem_raw[];
  T* smem = reinterpret_cast<T*>(smem_raw);

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int h = lane >> 5, c = lane & 31;

  const int w = xcd_remap(blockIdx.x, gridDim.x);
  const int qt_idx = w % p.n_qtiles;
  const int bh = bh_of_group(w / p.n_qtiles, p.bh, p.heads);
  const int qtile = CAUSAL ? (p.n_qtiles - 1 - qt_idx) : qt_idx;
  const int64_t q0 = (int64_t)qtile * BQ;
  const int64_t qw = q0 + 32 * QT * wave;  // first query of this wave

  const T* __restrict__ qg = static_cast<const T*>(p.q) + head_base(p.sq, bh, p.heads);
  const TO* __restrict__ dog = static_cast<const TO*>(p.d_o) + head_base(p.sdo, bh, p.heads);
  const T* __restrict__ kg = static_cast<const T*>(p.k) + head_base(p.sk, bh, p.heads);
  const T* __restrict__ vg = static_cast<const T*>(p.v) + head_base(p.sv, bh, p.heads);

  // Q^T and dO^T as B operands: lane (h, query c of sub-tile t), k = 16kc + 8h + s.
  // Initial values of the S^T and dP^T accumulators of each query: -lse/scale
  // (P = 2^(c*acc)) and -D (dS = P*acc); -inf for a padding row.
  Frag<T> qf[QT][KC], gf[QT][KCV];
  float s_init[QT], dp_init[QT];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const int64_t query = qw + 32 * t + c;
    const bool valid = query < p.n_q;
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
      if (valid) {
        qf[t][kc] = *reinterpret_cast<const Frag<T>*>(qg + query * p.sq.r + 16 * kc + 8 * h);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[t][kc][e] = (T)0.0f;
      }
    }
#pragma unroll
    for (int kc = 0; kc < KCV; ++kc) {
      if (valid) {
        gf[t][kc] = ld_frag_as<T, TO>(dog + query * p.sdo.r + 16 * kc + 8 * h);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) gf[t][kc][e] = (T)0.0f;
      }
    }
    s_init[t] = valid ? p.s_init[(size_t)bh * p.n_q_pad + query] : -INFINITY;
    dp_init[t] = valid ? p.dp_init[(size_t)bh * p.n_q_pad + query] : 0.0f;
  }
  wait_global_loads();

  f32x16 acc[QT][NDT];
#pragma unroll
  for (int t = 0; t < QT; ++t)
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[t][dt][r] = 0.0f;

  // Keys visible to this (batch, head): n_k, or the batch's valid length
  // (key padding); loads stay bounded by n_k.
  const int64_t n_kv = valid_keys(p.kv_len, bh, p.heads, p.n_k);
  int64_t ke = n_kv;
  if (CAUSAL && ke > q0 + BQ) ke = q0 + BQ;
  const int n_tiles = (int)((ke + BK - 1) / BK);

  // Register sets for the global -> LDS staging (see the dK/dV kernel): with
  // PF = 2 tile j + 2 is loaded while tile j + 1 is written to LDS.  Off
  // (PF = 1): with the causal early exit of a tile the compiler moved the
  // two sets to scratch memory and the kernel ran 5x slower.
  constexpr int PF = 1;
  u32x4 stage_a[CPT], stage_b[CPT];
  auto load_stage = [&](auto set_tag, int64_t k0) __attribute__((always_inline)) {
    u32x4 (&stage)[CPT] = decltype(set_tag)::value ? stage_b : stage_a;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      // The K tile's BK * CPRK chunks, then the V tile's.
      const int chunk = tid + i * NT;
      const bool is_v = chunk >= BK * CPRK;
      const int rem = is_v ? chunk - BK * CPRK : chunk;
      const int cpr = is_v ? CPRV : CPRK;
      const int row = rem / cpr, col = rem % cpr;
      const int64_t kr = k0 + row;
      const T* src = (is_v ? vg + kr * p.sv.r : kg + kr * p.sk.r) + col * (16 / E);
      stage[i] = kr < p.n_k ? ld16(src) : u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto store_stage = [&](auto set_tag, int buf) __attribute__((always_inline)) {
    const u32x4 (&stage)[CPT] = decltype(set_tag)::value ? stage_b : stage_a;
    T* base = smem + buf * (TILEK + TILEV);
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int chunk = tid + i * NT;
      const bool is_v = chunk >= BK * CPRK;
      const int rem = is_v ? chunk - BK * CPRK : chunk;
      const int cpr = is_v ? CPRV : CPRK;
      const int row = rem / cpr, col = rem % cpr;
      st16(base + (is_v ? TILEK + row * RSV : row * RSK) + col * (16 / E), stage[i]);
    }
  };

  // SWZ copies: a tile is 8 K units and 8 V units of 1 KiB (4 rows each);
  // wave w copies units w and w + 4 of both, i.e. rows 4w + lane / 16 and 16
  // rows further, which share their swizzle.  Full tiles take a scalar base
  // and per-lane byte offsets computed once; in a ragged last tile rows past
  // n_k copy row n_k - 1 (finite values whose weights are masked to 0).
  const int crow = 4 * wave + (lane >> 4);
  const int cchunk = (lane & 15) ^ swz128(crow);
  const unsigned koff = (unsigned)(crow * p.sk.r) * E + 16u * (unsigned)cchunk;
  const unsigned voff = (unsigned)(crow * p.sv.r) * E + 16u * (unsigned)cchunk;
  auto copy_tile = [&](int64_t k0, int buf) __attribute__((always_inline)) {
    const unsigned dst =
        __builtin_amdgcn_readfirstlane(lds_addr(smem + buf * (TK + TV)) + 1024u * (unsigned)wave);
    if (k0 + BK <= p.n_k) {
      const T* kb = kg + k0 * p.sk.r;
      const T* vb = vg + k0 * p.sv.r;
      copy_to_lds16_sb(kb, koff, dst);
      copy_to_lds16_sb(kb + 16 * p.sk.r, koff, dst + 4096u);
      copy_to_lds16_sb(vb, voff, dst + 8192u);
      copy_to_lds16_sb(vb + 16 * p.sv.r, voff, dst + 12288u);
    } else {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        int64_t kr = k0 + crow + 16 * j;
        if (kr > p.n_k - 1) kr = p.n_k - 1;
        copy_to_lds16(kg + kr * p.sk.r + 8 * cchunk, dst + 4096u * j);
        copy_to_lds16(vg + kr * p.sv.r + 8 * cchunk, dst + 8192u + 4096u * j);
      }
    }
  };

  const int krow = perm32(c);
  const float cl2 = p.scale_log2;

  if constexpr (SWZ) {
    if (n_tiles > 0) {
      copy_tile(0, 0);
      wait_global_loads();
    }
  } else {
    if (n_tiles > 0) {
      load_stage(BoolC<false>{}, 0);
      store_stage(BoolC<false>{}, 0);
    }
    if (PF == 2 && n_tiles > 1) load_stage(BoolC<true>{}, BK);
  }
  __syncthreads();

  // Leading tiles that need no mask (all keys exist and, causal, precede the
  // workgroup's first query); masked tiles run in a second loop.
  int n_plain = (int)(n_kv / BK);
  if (n_plain > n_tiles) n_plain = n_tiles;
  if (CAUSAL) {
    const int below = (int)((q0 + 1) / BK);
    if (below < n_plain) n_plain = below;
  }

  auto tile = [&](auto mask_tag, int it) {
    constexpr bool MASK = decltype(mask_tag)::value;
    const int64_t k0 = (int64_t)it * BK;
    const T* ks = smem + (it & 1) * (TK + TV);
    const T* vs = ks + TK;
    if (MASK && CAUSAL && k0 > qw + 32 * QT - 1) return;  // all keys after this wave's queries
    f32x16 s[NKT][QT], dp[NKT][QT];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int t = 0; t < QT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          s[kt][t][r] = s_init[t];
          dp[kt][t][r] = dp_init[t];
        }
    // S^T = K Q^T - lse/scale and dP^T = V dO^T - D (rows: keys in perm32
    // order; lane: query).
    if constexpr (SWZ && QT == 1 && NKT == 1 && DQ_AHEAD > 0) {
      // The K and V row fragments of k chunk kc are read DQ_AHEAD chunks
      // before their MFMAs (a ring of registers), so the MFMAs do not wait on
      // reads issued just before them.
      constexpr int RA = DQ_AHEAD + 1;
      Frag<T> fa[RA], fb[RA];
      auto fetch = [&](int kc) __attribute__((always_inline)) {
        fa[kc % RA] = lds_frag_swz128<T>(ks, krow, 2 * kc + h);
        fb[kc % RA] = lds_frag_swz128<T>(vs, krow, 2 * kc + h);
      };
#pragma unroll
      for (int kc = 0; kc < DQ_AHEAD; ++kc) fetch(kc);
#pragma unroll
      for (int kc = 0; kc < KC; ++kc) {
        if (kc + DQ_AHEAD < KC) fetch(kc + DQ_AHEAD);
        s[0][0] = mma(fa[kc % RA], qf[0][kc], s[0][0]);
        dp[0][0] = mma(fb[kc % RA], gf[0][kc], dp[0][0]);
        __builtin_amdgcn_sched_barrier(0);
      }
    } else
#pragma unroll
    for (int kc = 0; kc < (KC > KCV ? KC : KCV); ++kc)
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        if (kc < KC) {
          const Frag<T> a = SWZ ? lds_frag_swz128<T>(ks, 32 * kt + krow, 2 * kc + h)
                                : lds_frag<T>(ks + (32 * kt + krow) * RSK + 16 * kc + 8 * h);
#pragma unroll
          for (int t = 0; t < QT; ++t) s[kt][t] = mma(a, qf[t][kc], s[kt][t]);
        }
        if (kc < KCV) {
          const Frag<T> b = SWZ ? lds_frag_swz128<T>(vs, 32 * kt + krow, 2 * kc + h)
                                : lds_frag<T>(vs + (32 * kt + krow) * RSV + 16 * kc + 8 * h);
#pragma unroll
          for (int t = 0; t < QT; ++t) dp[kt][t] = mma(b, gf[t][kc], dp[kt][t]);
        }
      }
    // Tile-relative 32-bit bounds: key k0 + x is valid iff x < key_lim and,
    // under the causal mask, visible to query qw + 32t + c iff x <= q_rel + 32t.
    int key_lim = BK, q_rel = BK;
    if constexpr (MASK) {
      key_lim = (int)(n_kv - k0 < BK ? n_kv - k0 : BK);
      if (CAUSAL) q_rel = (int)(qw - k0) + c;
    }
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      int lim = key_lim;
      if (MASK && CAUSAL && q_rel + 32 * t + 1 < lim) lim = q_rel + 32 * t + 1;
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float pr = fast_exp2(s[kt][t][r] * cl2);
          if (MASK && 32 * kt + permuted_row(r, h) >= lim) pr = 0.0f;
          dp[kt][t][r] = pr * dp[kt][t][r];  // dS^T
        }
    }
    // dQ^T += K^T dS^T.
#pragma unroll
    for (int pc = 0; pc < NPC; ++pc) {
      Frag<T> b[QT];
#pragma unroll
      for (int t = 0; t < QT; ++t) {
        float td[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) td[e] = dp[pc >> 1][t][8 * (pc & 1) + e];
        b[t] = to_frag<T>(td);
      }
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        Frag<T> a;
        if constexpr (SWZ) {
          a = lds_col_frag_swz128<T>(ks, 16 * pc, 32 * dt, lane);
        } else if constexpr (sizeof(T) == 2) {
          a = lds_col_frag<T>(ks, RSK, 16 * pc, 32 * dt, lane);
        } else {
          a = lds_col_frag_f32(reinterpret_cast<const float*>(ks), RSK, 16 * pc, 32 * dt, lane);
        }
#pragma unroll
        for (int t = 0; t < QT; ++t) acc[t][dt] = mma(a, b[t], acc[t][dt]);
      }
    }
  };
  // Tile j is computed from LDS buffer j & 1 while tile j + 1 is written to
  // the other one.  PF = 2: set A holds even tiles, set B odd ones, and tile
  // j + 2 is loaded into the set that held tile j; PF = 1: tile j + 1 is
  // loaded into set A in this iteration.
  auto step = [&](auto mask_tag, auto odd_tag, int it) __attribute__((always_inline)) {
    constexpr bool ODD = decltype(odd_tag)::value;
    if constexpr (SWZ) {
      if (it + 1 < n_tiles) copy_tile((int64_t)(it + 1) * BK, (it + 1) & 1);
      tile(mask_tag, it);
      if (it + 1 < n_tiles) wait_global_loads();
      __syncthreads();
      return;
    }
    if constexpr (PF == 2) {
      if (it + 2 < n_tiles) load_stage(BoolC<ODD>{}, (int64_t)(it + 2) * BK);
    } else {
      if (it + 1 < n_tiles) load_stage(BoolC<false>{}, (int64_t)(it + 1) * BK);
    }
    tile(mask_tag, it);
    if (it + 1 < n_tiles) store_stage(BoolC<PF == 2 && !ODD>{}, (it + 1) & 1);
    __syncthreads();
  };
  auto run = [&](auto mask_tag, int it) __attribute__((always_inline)) {
    if (PF == 2 && (it & 1)) step(mask_tag, BoolC<true>{}, it);
    else step(mask_tag, BoolC<false>{}, it);
  };
  int it = 0;
  for (; it < n_plain; ++it) run(BoolC<false>{}, it);
  for (; it < n_tiles; ++it) run(BoolC<true>{}, it);

#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const int64_t query = qw + 32 * t + c;
    if (query >= p.n_q) continue;
    T* dqg = static_cast<T*>(p.dq) + head_base(p.sdq, bh, p.heads) + query * p.sdq.r;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int a4 = 0; a4 < 4; ++a4) {
        typename FragT<T>::half v4;
#pragma unroll
        for (int e = 0; e < 4; ++e) v4[e] = (T)(acc[t][dt][4 * a4 + e] * p.scale);
        *reinterpret_cast<typename FragT<T>::half*>(dqg + 32 * dt + 8 * a4 + 4 * h) = v4;
      }
  }
}

// ------------------------------------------------------- dQ (two groups)
// 16-bit inputs and outputs, d = 64.  Eight waves of 32 queries each (Q, dO
// and the accumulator initial values in registers, dQ accumulated in
// registers) in two groups of four that alternate an MFMA phase and a VALU
// phase like the two-group dK/dV kernel.  MFMA phase of key tile j:
// dQ^T += K^T dS^T for tile j - 1, then S^T = K Q^T and dP^T = V dO^T for
// tile j.  VALU phase: P = 2^(c S), dS = P dP, rounded into the operands of
// the next MFMA phase.  K and V stream through a four-stage LDS ring.
namespace qpp {
constexpr int D = 64, NW = 8, BQG = NW * 32, BK = 64, NKT = BK / 32, NSTAGE = MEA_T64_DQ_NSTAGE;
// Copy lead, in tiles, of group 1 and group 0 (see the copy schedule below).
constexpr int LEAD1 = NSTAGE - 1, LEAD0 = NSTAGE - 2;
static_assert(NSTAGE >= 4 && NSTAGE <= 6, "K/V stages");
constexpr int RSB = 144;                 // bytes per LDS row (128 + 16 pad)
constexpr int TILEB = BK * RSB;          // one K or V tile: 9 KiB
constexpr int STAGEB = 2 * TILEB;
constexpr int UNITS = 2 * TILEB / 1024;  // 1 KiB copies per stage (18)
static_assert(TILEB % 1024 == 0, "stage layout");
}  // namespace qpp

template <typename T, bool CAUSAL>
__global__ __launch_bounds__(512, 1) void attn_bwd_dq_pp_kernel(BwdParams p) {
  using namespace qpp;
  static_assert(sizeof(T) == 2, "16-bit inputs only");
  constexpr int KC = D / 16, NDT = D / 32, NPC = BK / 16;
  __shared__ __align__(16) unsigned char smem[NSTAGE * STAGEB];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2;
  const int lane = tid & 63;
  const int h = lane >> 5, c = lane & 31;

  const int w = xcd_remap(blockIdx.x, gridDim.x);
  const int qt_idx = w % p.n_qtiles;
  const int bh = bh_of_group(w / p.n_qtiles, p.bh, p.heads);
  const int qtile = CAUSAL ? (p.n_qtiles - 1 - qt_idx) : qt_idx;  // heaviest first
  const int64_t q0 = (int64_t)qtile * BQG;
  const int64_t qw = q0 + 32 * wave;  // first query of this wave
  const int64_t query = qw + c;

  const T* __restrict__ qg = static_cast<const T*>(p.q) + head_base(p.sq, bh, p.heads);
  const T* __restrict__ dog = static_cast<const T*>(p.d_o) + head_base(p.sdo, bh, p.heads);
  const T* __restrict__ kg = static_cast<const T*>(p.k) + head_base(p.sk, bh, p.heads);
  const T* __restrict__ vg = static_cast<const T*>(p.v) + head_base(p.sv, bh, p.heads);

  // Q^T and dO^T as B operands: lane (h, query c), k = 16 kc + 8 h + s.
  Frag<T> qf[KC], gf[KC];
  const bool valid = query < p.n_q;
#pragma unroll
  for (int kc = 0; kc < KC; ++kc) {
    if (valid) {
      qf[kc] = *reinterpret_cast<const Frag<T>*>(qg + query * p.sq.r + 16 * kc + 8 * h);
      gf[kc] = *reinterpret_cast<const Frag<T>*>(dog + query * p.sdo.r + 16 * kc + 8 * h);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        qf[kc][e] = (T)0.0f;
        gf[kc][e] = (T)0.0f;
      }
    }
  }
  // The query's initial values from its record (three bf16 parts each).
  float s_init = -INFINITY, dp_init = 0.0f;
  if (valid) {
    const bf16x8 r = __builtin_bit_cast(bf16x8, p.row_rec[(size_t)bh * p.n_q_pad + query]);
    s_init = ((float)r[0] + (float)r[1]) + (float)r[2];
    dp_init = ((float)r[4] + (float)r[5]) + (float)r[6];
  }
  wait_global_loads();

  f32x16 acc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[dt][r] = 0.0f;

  // Keys after the workgroup's last query are invisible to all of it (causal),
  // and so are keys past the batch's valid length (key padding); loads stay
  // bounded by n_k.
  const int64_t n_kv = valid_keys(p.kv_len, bh, p.heads, p.n_k);
  int64_t ke = n_kv;
  if (CAUSAL && ke > q0 + BQG) ke = q0 + BQG;
  const int n_tiles = (int)((ke + BK - 1) / BK);
  auto stage = [&](int j) { return smem + (j % NSTAGE) * STAGEB; };

  // Copy unit u (0 <= u < UNITS) of key tile j: units 0..8 are the K tile,
  // 9..17 the V tile (lane slot s = 64 (u % 9) + lane is row s / 9, 16-byte
  // chunk s % 9; chunk 8 is the row pad and gets a copy of chunk 7).  The
  // lane's byte offset within a tile is computed once per unit; a tile that
  // ends past n_k takes the clamped path, whose rows past n_k repeat the last
  // key (finite values; masked).
  const int n_full = (int)(n_kv / BK);  // tiles with no key past the valid length
  auto unit_row = [&](int u) { return (64 * (u % 9) + lane) / 9; };
  auto unit_col = [&](int u) {
    const int ch = (64 * (u % 9) + lane) % 9;
    return (unsigned)(16 * (ch < 8 ? ch : 7));
  };
  // Byte offset within a tile (row strides < 2^24 elements, checked on the host).
  auto unit_off = [&](int u) {
    const unsigned rsb = (unsigned)sizeof(T) * (unsigned)(u >= 9 ? p.sv.r : p.sk.r);
    return (unsigned)unit_row(u) * rsb + unit_col(u);
  };
  auto copy_unit = [&](int j, int u, unsigned off) __attribute__((always_inline)) {
    const int which = u >= 9, v9 = u - 9 * which;
    const T* g = which ? vg : kg;
    const int64_t rs = which ? p.sv.r : p.sk.r;
    const unsigned lds = __builtin_amdgcn_readfirstlane(lds_addr(stage(j) + which * TILEB + 1024 * v9));
    const int64_t k0 = (int64_t)j * BK;
    if (j < n_full) {
      copy_to_lds16_sb(g + k0 * rs, off, lds);
    } else {
      int64_t key = k0 + unit_row(u);
      if (key > p.n_k - 1) key = p.n_k - 1;
      copy_to_lds16(reinterpret_cast<const unsigned char*>(g + key * rs) + unit_col(u), lds);
    }
  };
  constexpr int MAXU = (UNITS + NW - 1) / NW;
  const int n_units = (UNITS - wave + NW - 1) / NW;
  unsigned uoff[MAXU];
#pragma unroll
  for (int k = 0; k < MAXU; ++k) {
    const int u = wave + NW * k;
    uoff[k] = u < UNITS ? unit_off(u) : 0u;
  }
  auto issue = [&](int j) __attribute__((always_inline)) {
    if (j < n_tiles) {
#pragma unroll
      for (int k = 0; k < MAXU; ++k)
        if (wave + NW * k < UNITS) copy_unit(j, wave + NW * k, uoff[k]);
    }
  };
  // Wait for this wave's copies of tile j + 1 while its copies of the tiles
  // after it, up to tile `last` (the newest issued), may still run.
  auto wait_copies = [&](int j, int last) __attribute__((always_inline)) {
    if (last > n_tiles - 1) last = n_tiles - 1;
    const int later = last - (j + 1);
    wait_global_loads_rt<3 * (LEAD1 - 2)>(later > 0 ? later * n_units : 0);
  };
  auto barrier = [&]() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" ::: "memory");
  };

  // Copy schedule: group 1 issues its share of tile j in its VALU phase of
  // tile j - LEAD1, group 0 in its VALU phase of tile j - LEAD0; both wait for
  // tile j before the barrier that precedes group 0's MFMA phase of tile j.
  // The last reader of tile j's stage is group 1's MFMA phase of tile j + 1
  // (the dQ steps of tile j), two phases before the VALU phase of group 1 that
  // overwrites it with tile j + NSTAGE and one before group 0's.
  if (n_tiles > 0)
    for (int u = wave; u < UNITS; u += NW) copy_unit(0, u, unit_off(u));
  wait_global_loads();
  __syncthreads();
  if (grp == 1) {
#pragma unroll
    for (int t = 1; t < LEAD1; ++t) issue(t);
    barrier();
  } else {
#pragma unroll
    for (int t = 1; t < LEAD0; ++t) issue(t);
  }

  const int krow = perm32(c);
  const float cl2 = p.scale_log2;
  f32x16 s[NKT], dp[NKT];
  Frag<T> dsf[NPC];
  // Whether tile j needs the elementwise mask (ragged keys, causal diagonal).
  auto masked = [&](int j) {
    const int64_t k0 = (int64_t)j * BK;
    return k0 + BK > n_kv || (CAUSAL && k0 + BK - 1 > qw);
  };
  constexpr int AHEAD = CAUSAL ? 2 : MEA_T64_DQ_AHEAD;
  // dQ^T += K^T dS^T for tile j (column fragments of K: k = keys).
  auto dq_mma = [&](int j) __attribute__((always_inline)) {
    const T* ks = reinterpret_cast<const T*>(stage(j));
    constexpr int NSTEP = NPC;
    Frag<T> ka[2][AHEAD + 1];
    auto fetch = [&](int step) __attribute__((always_inline)) {
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
        ka[dt][step % (AHEAD + 1)] = lds_col_frag<T>(ks, RSB / 2, 16 * step, 32 * dt, lane);
    };
#pragma unroll
    for (int step = 0; step < AHEAD; ++step) fetch(step);
#pragma unroll
    for (int step = 0; step < NSTEP; ++step) {
      if (step + AHEAD < NSTEP) fetch(step + AHEAD);
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) acc[dt] = mma(ka[dt][step % (AHEAD + 1)], dsf[step], acc[dt]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // S^T = K Q^T + s_init and dP^T = V dO^T + dp_init for tile j (row fragments).
  auto sdp = [&](int j) __attribute__((always_inline)) {
    const T* ks = reinterpret_cast<const T*>(stage(j));
    const T* vs = reinterpret_cast<const T*>(stage(j) + TILEB);
    constexpr int NSTEP = KC * NKT;
    Frag<T> fa[AHEAD + 1], fb[AHEAD + 1];
    auto fetch = [&](int step) __attribute__((always_inline)) {
      const int kc = step / NKT, kt = step % NKT;
      fa[step % (AHEAD + 1)] = lds_frag<T>(ks + (32 * kt + krow) * (RSB / 2) + 16 * kc + 8 * h);
      fb[step % (AHEAD + 1)] = lds_frag<T>(vs + (32 * kt + krow) * (RSB / 2) + 16 * kc + 8 * h);
    };
#pragma unroll
    for (int step = 0; step < AHEAD; ++step) fetch(step);
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[kt][r] = s_init;
        dp[kt][r] = dp_init;
      }
#pragma unroll
    for (int step = 0; step < NSTEP; ++step) {
      if (step + AHEAD < NSTEP) fetch(step + AHEAD);
      const int kc = step / NKT, kt = step % NKT;
      s[kt] = mma(fa[step % (AHEAD + 1)], qf[kc], s[kt]);
      dp[kt] = mma(fb[step % (AHEAD + 1)], gf[kc], dp[kt]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // Keys of tile j visible to the wave's queries, for the masked variants:
  // key k0 + x is valid iff x < lim (ragged tail; causal: x <= query - k0).
  auto key_lim = [&](int j) {
    const int64_t k0 = (int64_t)j * BK;
    int lim = (int)(n_kv - k0 < BK ? n_kv - k0 : BK);
    if (CAUSAL) {
      const int64_t qr = query - k0 + 1;
      if (qr < lim) lim = qr > 0 ? (int)qr : 0;
    }
    return lim;
  };
  // P = 2^(c S), dS = P dP for four keys of 16-key chunk pc (half hf of it),
  // rounded and packed into two dwords of the chunk's dS^T operand.
  auto pds_half = [&](auto mask_tag, int pc, int hf, int lim) __attribute__((always_inline)) {
    constexpr bool MASK = decltype(mask_tag)::value;
    const int kt = pc >> 1;
    float ds[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = 8 * (pc & 1) + 4 * hf + e;
      float pr = fast_exp2(s[kt][r] * cl2);
      if (MASK && 32 * kt + permuted_row(r, h) >= lim) pr = 0.0f;
      ds[e] = pr * dp[kt][r];
    }
    return u32x2{pack2<T>(ds[0], ds[1]), pack2<T>(ds[2], ds[3])};
  };
  // Chunks pc0 .. NPC - 1 of tile j (the softmax phase's share), in groups of
  // G keys per lane whose multiplies, exponentials, multiplies and conversions
  // are issued as separate stages: G independent chains per stage hide the
  // latency of each stage behind the issue of the next (the compiler would
  // otherwise reuse a few temporaries and serialise short chains).
  auto pds = [&](auto mask_tag, int pc0, int lim) __attribute__((always_inline)) {
    constexpr bool MASK = decltype(mask_tag)::value;
    constexpr int G = MEA_T64_DQ_G;
    static_assert(G == 8 || G == 16, "8 or 16 keys per lane per group");
#pragma unroll
    for (int g0 = 8 * pc0; g0 < 8 * NPC; g0 += G) {
      const int n = 8 * NPC - g0 < G ? 8 * NPC - g0 : G;
      float x[G];
#pragma unroll
      for (int e = 0; e < n; ++e) x[e] = s[(g0 + e) >> 4][(g0 + e) & 15] * cl2;
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int e = 0; e < n; ++e) {
        x[e] = fast_exp2(x[e]);
        const int kt = (g0 + e) >> 4, r = (g0 + e) & 15;
        if (MASK && 32 * kt + permuted_row(r, h) >= lim) x[e] = 0.0f;
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int e = 0; e < n; ++e) x[e] *= dp[(g0 + e) >> 4][(g0 + e) & 15];
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int c8 = 0; c8 < n; c8 += 8) {
        dsf[(g0 + c8) >> 3] = to_frag<T>(x + c8);
        keep_here(dsf[(g0 + c8) >> 3]);  // the conversions belong to this phase
      }
    }
  };

  // MFMA phase of key tile j with dQ of tile j - 1 (steady state).  Steps, two
  // MFMAs each: 0..3 S^T/dP^T of keys 0..31 of tile j (k chunk = step), 4..7
  // dQ^T += K^T dS^T of tile j - 1 (key chunk = step - 4), 8..11 S^T/dP^T of
  // keys 32..63.  The first W 16-key chunks of tile j's dS (keys 0..31 are
  // final after step 3) are computed here, four keys per lane at a time
  // between the two MFMAs of a step, spread over steps 4..11; chunk pc is
  // written only after dQ step 4 + pc has read the old chunk pc.  One LDS
  // fetch ring runs through all twelve steps.
  constexpr int W = MEA_T64_DQ_W;
  static_assert(W >= 0 && W <= 2, "only chunks of keys 0..31 are final before the dQ steps");
  auto mfma_phase = [&](auto mask_tag, int j) __attribute__((always_inline)) {
    constexpr int NS = 12;
    const T* ks = reinterpret_cast<const T*>(stage(j));
    const T* vs = reinterpret_cast<const T*>(stage(j) + TILEB);
    const T* kp = reinterpret_cast<const T*>(stage(j - 1));
    Frag<T> rx[AHEAD + 1], ry[AHEAD + 1];
    auto fetch = [&](int g) __attribute__((always_inline)) {
      const int slot = g % (AHEAD + 1);
      if (g >= 4 && g < 8) {
        rx[slot] = lds_col_frag<T>(kp, RSB / 2, 16 * (g - 4), 0, lane);
        ry[slot] = lds_col_frag<T>(kp, RSB / 2, 16 * (g - 4), 32, lane);
      } else {
        const int kt = g >= 8, kc = g - 8 * kt;
        rx[slot] = lds_frag<T>(ks + (32 * kt + krow) * (RSB / 2) + 16 * kc + 8 * h);
        ry[slot] = lds_frag<T>(vs + (32 * kt + krow) * (RSB / 2) + 16 * kc + 8 * h);
      }
    };
    const int lim = decltype(mask_tag)::value ? key_lim(j) : BK;
#pragma unroll
    for (int g = 0; g < AHEAD; ++g) fetch(g);
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[kt][r] = s_init;
        dp[kt][r] = dp_init;
      }
    u32x2 first_half = {0u, 0u};
#pragma unroll
    for (int g = 0; g < NS; ++g) {
      if (g + AHEAD < NS) fetch(g + AHEAD);
      const int slot = g % (AHEAD + 1);
      // Half-chunk u of the dS work runs in step 4 + (4 u) / W.
      int u = -1;
      if constexpr (W > 0) {
#pragma unroll
        for (int uu = 0; uu < 2 * W; ++uu)
          if (g == 4 + (4 * uu) / W) u = uu;
      }
      if (g >= 4 && g < 8) {
        acc[0] = mma(rx[slot], dsf[g - 4], acc[0]);
      } else {
        const int kt = g >= 8, kc = g - 8 * kt;
        s[kt] = mma(rx[slot], qf[kc], s[kt]);
      }
      if (u >= 0) {
        const u32x2 part = pds_half(mask_tag, u >> 1, u & 1, lim);
        if ((u & 1) == 0) first_half = part;
        else dsf[u >> 1] = __builtin_bit_cast(Frag<T>, u32x4{first_half[0], first_half[1], part[0], part[1]});
      }
      if (g >= 4 && g < 8) {
        acc[1] = mma(ry[slot], dsf[g - 4], acc[1]);
      } else {
        const int kt = g >= 8, kc = g - 8 * kt;
        dp[kt] = mma(ry[slot], gf[kc], dp[kt]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // One iteration per key tile.  MODE 1: the first tile (S/dP only); MODE 2:
  // dQ of the previous tile and S/dP of this one; MODE 3: dQ of the previous
  // tile only (this one is past the wave's last query, causal); MODE 0:
  // copies and barriers only.  A tile past the wave's last query stays so for
  // the later tiles (the keys only grow), so the modes come in this order and
  // each loop below runs one of them; MODE 2 runs unmasked tiles, then masked
  // ones (ragged tail, causal diagonal), which also come last.
  auto iteration = [&](auto mode_tag, auto mask_tag, int j) __attribute__((always_inline)) {
    constexpr int MODE = decltype(mode_tag)::value;
    constexpr bool MASK = decltype(mask_tag)::value;
    // ---- MFMA phase
    mfma_phase_priority();
    if constexpr (MODE == 2) mfma_phase(mask_tag, j);
    if constexpr (MODE == 3) dq_mma(j - 1);
    if constexpr (MODE == 1) sdp(j);
    if (grp == 1) wait_copies(j, j - 1 + LEAD1);
    barrier();
    // ---- VALU phase
    valu_phase_priority();
    if constexpr (MODE == 1) {
      if (masked(j)) pds(BoolC<true>{}, 0, key_lim(j));
      else pds(BoolC<false>{}, 0, BK);
    } else if constexpr (MODE == 2) {
      pds(mask_tag, W, MASK ? key_lim(j) : BK);
    }
    if (grp == 1) {
      issue(j + LEAD1);
    } else {
      issue(j + LEAD0);
      wait_copies(j, j + LEAD0);
    }
    barrier();
  };
  // Tiles 0 .. j_end - 1 hold keys visible to the wave; tiles j_mask and
  // later need the elementwise mask.
  int j_end = n_tiles;
  int j_mask = n_full;
  if (CAUSAL) {
    const int64_t last = (qw + 31) / BK + 1;
    if (last < j_end) j_end = (int)last;
    // tile j holds a key after query qw iff 64 j + 63 > qw
    const int jc = qw < BK - 1 ? 0 : (int)((qw - (BK - 1)) / BK) + 1;
    if (jc < j_mask) j_mask = jc;
  }
  int j = 0;
  if (j < j_end) iteration(IntC<1>{}, BoolC<false>{}, j++);
  for (; j < j_end && j < j_mask; ++j) iteration(IntC<2>{}, BoolC<false>{}, j);
  for (; j < j_end; ++j) iteration(IntC<2>{}, BoolC<true>{}, j);
  if (j < n_tiles) iteration(IntC<3>{}, BoolC<false>{}, j++);
  for (; j < n_tiles; ++j) iteration(IntC<0>{}, BoolC<false>{}, j);
  if (j_end == n_tiles && n_tiles > 0) dq_mma(n_tiles - 1);
  if (grp == 0) barrier();  // group 1's start delay, balanced

  if (valid) {
    T* dqg = static_cast<T*>(p.dq) + head_base(p.sdq, bh, p.heads) + query * p.sdq.r;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int a4 = 0; a4 < 4; ++a4) {
        typename FragT<T>::half v4;
#pragma unroll
        for (int e = 0; e < 4; ++e) v4[e] = (T)(acc[dt][4 * a4 + e] * p.scale);
        *reinterpret_cast<typename FragT<T>::half*>(dqg + 32 * dt + 8 * a4 + 4 * h) = v4;
      }
  }
}

// ---------------------------------------------------------------- launchers

// Tile choices.  dK/dV: QS query sub-tiles of 32 per stage; dQ: QT query
// sub-tiles of 32 per wave and BK keys per stage; OCC = workgroups per CU the
// register budget is sized for.  The d = 64 16-bit choices can be overridden
// at build time for tuning sweeps.
#ifndef MEA_T64_DKDV_QS
#define MEA_T64_DKDV_QS 2
#endif
#ifndef MEA_T64_DKDV_OCC
#define MEA_T64_DKDV_OCC 2
#endif
#ifndef MEA_T64_DQ_QT
#define MEA_T64_DQ_QT 1
#endif
#ifndef MEA_T64_DQ_BK
#define MEA_T64_DQ_BK 64
#endif
#ifndef MEA_T64_DQ_OCC
#define MEA_T64_DQ_OCC 2
#endif
template <typename T, int D> struct BwdShape;
template <> struct BwdShape<__bf16, 64> {
  static constexpr int QS = MEA_T64_DKDV_QS, KV_OCC = MEA_T64_DKDV_OCC;
  static constexpr int QT = MEA_T64_DQ_QT, BK = MEA_T64_DQ_BK, Q_OCC = MEA_T64_DQ_OCC;
};
// d = 128, 16-bit: two workgroups per CU, whose waves overlap each other's
// MFMA, softmax and LDS work.  dK/dV fits them by keeping each lane's K
// fragments in LDS (K, V, dK and dV of 32 keys in registers would not fit;
// 25 % less time than one workgroup per CU), dQ by using 32-key tiles (37 %
// less time than 64-key tiles at one workgroup per CU).
#ifndef MEA_T128_DKDV_OCC
#define MEA_T128_DKDV_OCC 2
#endif
template <> struct BwdShape<__bf16, 128> {
  static constexpr int QS = 1, KV_OCC = MEA_T128_DKDV_OCC, QT = 1, BK = 32, Q_OCC = 2;
};
template <> struct BwdShape<_Float16, 64> : BwdShape<__bf16, 64> {};
template <> struct BwdShape<_Float16, 128> : BwdShape<__bf16, 128> {};
template <> struct BwdShape<float, 64> {
  static constexpr int QS = 2, KV_OCC = 1, QT = 1, BK = 32, Q_OCC = 2;
};
template <> struct BwdShape<float, 128> {
  static constexpr int QS = 1, KV_OCC = 1, QT = 1, BK = 32, Q_OCC = 1;
};

// dK/dV, then dQ (the per-row values already written by the preprocess);
// pp: the two-group kernels (which the caller has checked the layout for).
template <typename T, typename TO, int D, int DV, bool CAUSAL>
static hipError_t launch_bwd_kernels(BwdParams p, bool pp, hipStream_t stream) {
  using S = BwdShape<T, (D > DV ? D : DV)>;
  using Dk = DkdvTile<T, D, DV, S::QS>;
  void* args[] = {&p};
  constexpr bool PP_CAN = bwd_two_group_exists(sizeof(T) == 2, D, DV, __is_same(T, TO));
  hipError_t e = hipSuccess;
  if (p.dk) {
    bool launched = false;
    if constexpr (PP_CAN) {
      if (pp) {
        p.n_ktiles = (int)((p.n_k + kvpp::BKG - 1) / kvpp::BKG);
        e = hipLaunchKernel(reinterpret_cast<const void*>(attn_bwd_dkdv_pp_kernel<T, CAUSAL>),
                            dim3((unsigned)((int64_t)p.n_ktiles * p.bh)), dim3(kvpp::NW * 64), args, 0, stream);
        launched = true;
      }
    }
    if (!launched) {
      p.n_ktiles = (int)((p.n_k + Dk::BKG - 1) / Dk::BKG);
      e = hipLaunchKernel(reinterpret_cast<const void*>(attn_bwd_dkdv_kernel<T, TO, D, DV, S::QS, S::KV_OCC, CAUSAL>),
                          dim3((unsigned)((int64_t)p.n_ktiles * p.bh)), dim3(256), args,
                          Dk::lds_bytes(S::KV_OCC, __is_same(T, TO)), stream);
    }
    if (e != hipSuccess || !p.dq) return e;
  }
  if constexpr (PP_CAN) {
    if (pp) {
      p.n_qtiles = (int)((p.n_q + qpp::BQG - 1) / qpp::BQG);
      return hipLaunchKernel(reinterpret_cast<const void*>(attn_bwd_dq_pp_kernel<T, CAUSAL>),
                             dim3((unsigned)((int64_t)p.n_qtiles * p.bh)), dim3(qpp::NW * 64), args, 0, stream);
    }
  }
  p.n_qtiles = (int)((p.n_q + 128 * S::QT - 1) / (128 * S::QT));
  const int dq_lds = 2 * S::BK * (D + DV + 2 * 16 / (int)sizeof(T)) * (int)sizeof(T);
  return hipLaunchKernel(reinterpret_cast<const void*>(attn_bwd_dq_kernel<T, TO, D, DV, S::QT, S::BK, S::Q_OCC, CAUSAL>),
                         dim3((unsigned)((int64_t)p.n_qtiles * p.bh)), dim3(256), args, dq_lds, stream);
}

// D: head dimension of q and k; DV: of v, o and dO (tile shapes of the
// larger of the two).
template <typename T, typename TO, int D, int DV, bool CAUSAL>
static hipError_t launch_bwd_impl(BwdParams p, hipStream_t stream) {
  void* args[] = {&p};
  const int64_t rows = (int64_t)p.bh * p.n_q_pad;
  constexpr int RPB = 256 / (DV * (int)sizeof(TO) / 16);
  if constexpr (sizeof(T) == 2 && !__is_same(T, TO)) {
    if (p.do16) {
      // Float32 o and dO with 16-bit inputs: the preprocess also writes dO
      // rounded to T (the rounding the staging of these kernels applies), and
      // the kernels of 16-bit outputs run on that copy.
      constexpr bool PP_CAN = bwd_two_group_exists(true, D, DV, true);
      const bool pp = PP_CAN && bwd_two_group(true, D, DV, true, CAUSAL, p.n_q);
      if (pp ? p.row_rec == nullptr : (p.s_init == nullptr || p.dp_init == nullptr)) return hipErrorInvalidValue;
      const void* pre = reinterpret_cast<const void*>(attn_bwd_pre_kernel<TO, DV, false, T>);
      if constexpr (PP_CAN) {
        if (pp) pre = reinterpret_cast<const void*>(attn_bwd_pre_kernel<TO, DV, true, T>);
      }
      const hipError_t e = hipLaunchKernel(pre, dim3((unsigned)((rows + RPB - 1) / RPB)), dim3(256), args, 0, stream);
      if (e != hipSuccess) return e;
      BwdParams p16 = p;
      p16.d_o = p.do16;
      p16.sdo = TensorStrides{(int64_t)p.heads * p.n_q * DV, p.n_q * DV, DV};
      return launch_bwd_kernels<T, T, D, DV, CAUSAL>(p16, pp, stream);
    }
  }
  // The two-group kernels exist for 16-bit d = d_v = 64 with dO in the input
  // dtype; whether they run is the shared predicate's choice.
  constexpr bool PP_CAN = bwd_two_group_exists(sizeof(T) == 2, D, DV, __is_same(T, TO));
  const bool pp = PP_CAN && bwd_two_group(true, D, DV, true, CAUSAL, p.n_q);
  // The per-row values must be laid out as these kernels read them (records
  // or two arrays): a plan that disagrees is refused, not launched.
  if (pp ? p.row_rec == nullptr : (p.s_init == nullptr || p.dp_init == nullptr)) return hipErrorInvalidValue;
  const void* pre = reinterpret_cast<const void*>(attn_bwd_pre_kernel<TO, DV, false>);
  if constexpr (PP_CAN) {
    if (pp) pre = reinterpret_cast<const void*>(attn_bwd_pre_kernel<TO, DV, true>);
  }
  const hipError_t e = hipLaunchKernel(pre, dim3((unsigned)((rows + RPB - 1) / RPB)), dim3(256), args, 0, stream);
  if (e != hipSuccess) return e;
  return launch_bwd_kernels<T, TO, D, DV, CAUSAL>(p, pp, stream);
}

template <typename T, typename TO, int D, int DV = D>
static hipError_t launch_bwd_dt(const BwdParams& p, bool causal, hipStream_t stream) {
  return causal ? launch_bwd_impl<T, TO, D, DV, true>(p, stream) : launch_bwd_impl<T, TO, D, DV, false>(p, stream);
}

template <typename T, int D>
static hipError_t launch_bwd_out(const BwdParams& p, bool causal, bool out_f32, hipStream_t stream) {
  return out_f32 ? launch_bwd_dt<T, float, D>(p, causal, stream) : launch_bwd_dt<T, T, D>(p, causal, stream);
}

// Value head dimension different from the query/key one (64 and 128).
template <typename T, typename TO>
static hipError_t launch_bwd_dv_pair(const BwdParams& p, int d, bool causal, hipStream_t stream) {
  return d == 64 ? launch_bwd_dt<T, TO, 64, 128>(p, causal, stream) : launch_bwd_dt<T, TO, 128, 64>(p, causal, stream);
}

hipError_t launch_bwd(const BwdParams& p, int dtype, int d, int dv, bool causal, bool out_f32,
                      hipStream_t stream) {
  if (dv != d) {
    switch (dtype) {
      case 0: return launch_bwd_dv_pair<float, float>(p, d, causal, stream);
      case 1: return out_f32 ? launch_bwd_dv_pair<_Float16, float>(p, d, causal, stream)
                             : launch_bwd_dv_pair<_Float16, _Float16>(p, d, causal, stream);
      case 2: return out_f32 ? launch_bwd_dv_pair<__bf16, float>(p, d, causal, stream)
                             : launch_bwd_dv_pair<__bf16, __bf16>(p, d, causal, stream);
      default: return hipErrorInvalidValue;
    }
  }
  switch (dtype * 1000 + d) {
    case 0 * 1000 + 64: return launch_bwd_dt<float, float, 64>(p, causal, stream);
    case 0 * 1000 + 128: return launch_bwd_dt<float, float, 128>(p, causal, stream);
    case 1 * 1000 + 64: return launch_bwd_out<_Float16, 64>(p, causal, out_f32, stream);
    case 1 * 1000 + 128: return launch_bwd_out<_Float16, 128>(p, causal, out_f32, stream);
    case 2 * 1000 + 64: return launch_bwd_out<__bf16, 64>(p, causal, out_f32, stream);
    case 2 * 1000 + 128: return launch_bwd_out<__bf16, 128>(p, causal, out_f32, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace mea
