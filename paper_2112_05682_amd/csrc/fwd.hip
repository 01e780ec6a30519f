// Forward kernel: exact softmax attention over key/value tiles with the lazy
// softmax (arXiv 2112.05682, Eq. 1 of Section 2) made stable by the running
// maximum of Section 3, applied per tile of keys instead of per key:
//   m' = max(m, max_j s_j);  a = e^{m - m'};
//   l  <- a l + sum_j e^{s_j - m'};   acc <- a acc + sum_j e^{s_j - m'} v_j;
// and one division acc / l at the end.  Queries are tiled over workgroups
// (the query chunking of Section 4); the key loop is the Section 4 key-chunk
// loop with the summaries folded into the running state as they are made.
// With several key splits per query tile, each split writes its
// unnormalised summary (acc, m, l) and the combine kernel performs the
// Section 4 rescale-to-global-max, sum and divide.
//
// Work decomposition (gfx950, wave64, 32x32 MFMA tiles):
//   - a workgroup is 4 waves; each wave owns QT tiles of 32 queries, so a
//     workgroup covers BQ = 128*QT queries;
//   - K and V tiles of BK keys are staged through double-buffered LDS with
//     coalesced 16-byte global loads; Q stays in registers;
//   - scores are computed transposed, S^T = K Q^T, so that each lane owns one
//     query (column) and its softmax state is a per-lane scalar; the key rows
//     are read in the perm32 order so that the S^T tile, exponentiated and
//     rounded, is directly the B operand of O^T += V^T P^T;
//   - row max / row sum: in-lane over 16 registers, then one permlane32 swap
//     (the two lane halves hold disjoint keys of the same query);
//   - exp via v_exp_f32 (2^x) with scale*log2(e) folded into one FMA.
#include "device.hpp"
#include "kernels.hpp"

namespace mea {

constexpr float kLn2 = 0.6931471805599453f;

template <bool B> struct BoolC { static constexpr bool value = B; };
template <int I> struct IntC { static constexpr int value = I; };

// D: head dimension of q and k; DV: of v and o.
template <typename T, int D, int DV, int QT, int BK>
struct FwdTile {
  static constexpr int NW = 4;
  static constexpr int NT = NW * 64;
  static constexpr int BQ = NW * QT * 32;
  static constexpr int E = sizeof(T);
  // LDS row strides (elements).  K rows (read 16 bytes per lane, 16 rows
  // per 16 lanes) carry a 16-byte pad: each row starts 4 banks after the
  // previous one, so the 16 rows cover all 64 banks.  V rows are read by the
  // transposing read, 4 consecutive rows x 64 bytes per 32 lanes: a 64-byte pad
  // (16 banks) keeps those 4 rows in disjoint banks (a 16-byte pad made them
  // overlap 4 ways).  float32 V is read by scalar loads and keeps 16 bytes.
  static constexpr int RSK = D + 16 / E;
  static constexpr int RSV = DV + (E == 2 ? 64 : 16) / E;
  static constexpr int TILEK = BK * RSK;         // elements of the K tile
  static constexpr int TILEV = BK * RSV;         // elements of the V tile
  static constexpr int STAGE = TILEK + TILEV;    // one K/V stage
  static constexpr int CPRK = D * E / 16;        // 16-byte chunks per row
  static constexpr int CPRV = DV * E / 16;
  static constexpr int CHUNKS = BK * (CPRK + CPRV);  // K and V chunks per stage
  static constexpr int CPT = CHUNKS / NT;        // chunks per thread per stage
  static constexpr int LDS_BYTES = 2 * STAGE * E;  // double-buffered K and V
  static_assert(CHUNKS % NT == 0, "tile must split evenly over the workgroup");
  static_assert(BK % 32 == 0 && D % 32 == 0 && DV % 32 == 0, "tile shapes are multiples of 32");
};

#ifndef MEA_FWD_ILV
#define MEA_FWD_ILV 1
#endif
template <typename T, typename TO, int D, int DV, int QT, int BK, int OCC, bool CAUSAL>
__global__ __launch_bounds__(256, OCC) void attn_fwd_kernel(FwdParams p) {
  using Cfg = FwdTile<T, D, DV, QT, BK>;
  constexpr int RSK = Cfg::RSK, RSV = Cfg::RSV;
  constexpr int KC = D / 16;    // 16-wide k chunks of the QK^T contraction
  constexpr int NKT = BK / 32;  // 32-key sub-tiles per tile
  constexpr int NPC = BK / 16;  // 16-key chunks of the PV contraction
  constexpr int NDT = DV / 32;  // 32-row tiles of O^T
  constexpr bool ILV = MEA_FWD_ILV && sizeof(T) == 2 && NDT == 2;

  extern __shared__ __align__(16) unsigned char smem_raw[];
  T* smem = reinterpret_cast<T*>(smem_raw);

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int h = lane >> 5, c = lane & 31;

  // ---- workgroup -> (split, bh, query tile); heaviest causal tiles first.
  const int w = xcd_remap(blockIdx.x, gridDim.x);
  const int qt_idx = w % p.n_qtiles;
  const int rest = w / p.n_qtiles;
  const int bh = bh_of_group(rest % p.bh, p.bh, p.heads);
  const int split = rest / p.bh;
  const int qtile = CAUSAL ? (p.n_qtiles - 1 - qt_idx) : qt_idx;
  const int64_t q0 = (int64_t)qtile * Cfg::BQ;
  const int64_t qw = q0 + (int64_t)wave * QT * 32;  // first query of this wave

  const T* __restrict__ qg = static_cast<const T*>(p.q) + head_base(p.sq, bh, p.heads);
  const T* __restrict__ kg = static_cast<const T*>(p.k) + head_base(p.sk, bh, p.heads);
  const T* __restrict__ vg = static_cast<const T*>(p.v) + head_base(p.sv, bh, p.heads);

  // Keys visible to this (batch, head): n_k, or the batch's valid length.
  const int64_t n_k = valid_keys(p.kv_len, bh, p.heads, p.n_k);
  const int64_t kb = (int64_t)split * p.keys_per_split;
  int64_t ke = kb + p.keys_per_split;
  if (ke > n_k) ke = n_k;
  if (CAUSAL && ke > q0 + Cfg::BQ) ke = q0 + Cfg::BQ;  // keys beyond the last query are masked
  const int n_tiles = ke > kb ? (int)((ke - kb + BK - 1) / BK) : 0;

  // ---- Q fragments (B operand of S^T = K Q^T), resident for the whole loop.
  Frag<T> qf[QT][KC];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const int64_t row = qw + 32 * t + c;
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
      if (row < p.n_q) {
        qf[t][kc] = *reinterpret_cast<const Frag<T>*>(qg + row * p.sq.r + 16 * kc + 8 * h);
      } else {
#pragma unroll
        for (int s = 0; s < 8; ++s) qf[t][kc][s] = (T)0.0f;
      }
    }
  }

  wait_global_loads();

  f32x16 acc[QT][NDT];
#pragma unroll
  for (int t = 0; t < QT; ++t)
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[t][dt][r] = 0.0f;
  // Reference maximum (in units of scale * log2 e) and denominator per
  // query; each lane half accumulates the denominator of its own keys.
  float m_ref[QT], l_run[QT];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    m_ref[t] = -INFINITY;
    l_run[t] = 0.0f;
  }

  // ---- global -> register staging of one K/V stage (zero rows past n_k).
  u32x4 stage[Cfg::CPT];
  // Chunk i of a stage: the K tile's BK * CPRK chunks, then the V tile's.
  auto load_stage = [&](int64_t k0) {
#pragma unroll
    for (int i = 0; i < Cfg::CPT; ++i) {
      const int chunk = tid + i * Cfg::NT;
      const bool is_v = chunk >= BK * Cfg::CPRK;
      const int rem = is_v ? chunk - BK * Cfg::CPRK : chunk;
      const int cpr = is_v ? Cfg::CPRV : Cfg::CPRK;
      const int row = rem / cpr, col = rem % cpr;
      const int64_t key = k0 + row;
      const T* src = is_v ? vg + key * p.sv.r : kg + key * p.sk.r;
      src += col * (16 / Cfg::E);
      stage[i] = key < p.n_k ? ld16(src) : u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto store_stage = [&](int buf) {
    T* base = smem + buf * Cfg::STAGE;
#pragma unroll
    for (int i = 0; i < Cfg::CPT; ++i) {
      const int chunk = tid + i * Cfg::NT;
      const bool is_v = chunk >= BK * Cfg::CPRK;
      const int rem = is_v ? chunk - BK * Cfg::CPRK : chunk;
      const int cpr = is_v ? Cfg::CPRV : Cfg::CPRK;
      const int row = rem / cpr, col = rem % cpr;
      st16(base + (is_v ? Cfg::TILEK + row * RSV : row * RSK) + col * (16 / Cfg::E), stage[i]);
    }
  };

  const int krow = perm32(c);  // key row this lane feeds into the A operand
  const float cl2 = p.scale_log2;

  // Number of leading tiles that need no mask: every key exists (no ragged
  // tail) and, under the causal mask, precedes the workgroup's first query.
  int n_plain = n_tiles;
  {
    const int64_t full = n_k > kb ? (n_k - kb) / BK : 0;
    if (full < n_plain) n_plain = (int)full;
    if (CAUSAL) {
      const int64_t below = q0 - kb + 1 > 0 ? (q0 - kb + 1) / BK : 0;
      if (below < n_plain) n_plain = (int)below;
    }
  }

  // One K/V tile (LDS stage it & 1): S^T = K Q^T, (mask), online softmax with a
  // lazily raised reference maximum, O^T += V^T P^T.
  auto tile = [&](auto mask_tag, int it) {
    constexpr bool MASK = decltype(mask_tag)::value;
    const int64_t k0 = kb + (int64_t)it * BK;
    const T* ks = smem + (it & 1) * Cfg::STAGE;
    const T* vs = ks + Cfg::TILEK;
    // A wave whose queries all precede the tile's first key has nothing to do.
    if (MASK && CAUSAL && k0 > qw + QT * 32 - 1) return;

    f32x16 s[NKT][QT];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int t = 0; t < QT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[kt][t][r] = 0.0f;
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        const Frag<T> a = lds_frag<T>(ks + (32 * kt + krow) * RSK + 16 * kc + 8 * h);
#pragma unroll
        for (int t = 0; t < QT; ++t) s[kt][t] = mma(a, qf[t][kc], s[kt][t]);
      }
    }

    if constexpr (MASK) {
      // Tile-relative 32-bit bounds: key k0 + x is valid iff x < key_lim and,
      // under the causal mask, visible to query qw + 32t + c iff x <= q_rel + 32t.
      const int key_lim = (int)(n_k - k0 < BK ? n_k - k0 : BK);
      const int q_rel = CAUSAL ? (int)(qw - k0) + c : BK;
#pragma unroll
      for (int t = 0; t < QT; ++t) {
        const int lim_c = q_rel + 32 * t + 1;
        const int lim = CAUSAL && lim_c < key_lim ? lim_c : key_lim;
#pragma unroll
        for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (32 * kt + permuted_row(r, h) >= lim) s[kt][t][r] = -INFINITY;
      }
    }

    // Online softmax, one query per lane.  The reference maximum m_ref (kept
    // pre-multiplied by scale*log2 e) is raised only when a score exceeds it by
    // more than kRescaleSlack powers of two: weights stay <= 2^kRescaleSlack,
    // numerator and denominator share the reference, so the result is the same
    // and the accumulator rescale is skipped on most tiles.
    Frag<T> pf[QT][NPC];
    float neg[QT];
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kt][t][r]);
      const float mx_c = xhalf_max(mx) * cl2;
      const bool raise = mx_c > m_ref[t] + kRescaleSlack;
      if (__builtin_amdgcn_ballot_w64(raise)) {
        const float m_new = raise ? mx_c : m_ref[t];
        // 0 on a first raise; 1 for a lane that does not raise (also one still
        // at -inf, where the difference would be NaN).
        const float alpha = raise ? fast_exp2(m_ref[t] - m_new) : 1.0f;
        l_run[t] *= alpha;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[t][dt][r] *= alpha;
        m_ref[t] = m_new;
      }
      // A row with no visible key so far keeps m_ref = -inf; offset 0 keeps
      // its (all -inf) exponents at weight 0 instead of NaN.
      neg[t] = (MASK && m_ref[t] == -INFINITY) ? 0.0f : -m_ref[t];
#pragma unroll
      for (int pc = 0; pc < (ILV ? 1 : NPC); ++pc) {
        float e8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) e8[e] = fast_exp2(fmaf(s[pc >> 1][t][8 * (pc & 1) + e], cl2, neg[t]));
        pf[t][pc] = to_frag<T>(e8);
        l_run[t] = tree_sum<8>(e8, l_run[t]);
      }
    }
    auto col_v = [&](int pc, int dt) __attribute__((always_inline)) {
      if constexpr (sizeof(T) == 2) return lds_col_frag<T>(vs, RSV, 16 * pc, 32 * dt, lane);
      else return lds_col_frag_f32(reinterpret_cast<const float*>(vs), RSV, 16 * pc, 32 * dt, lane);
    };
    if constexpr (ILV) {
      // O^T += V^T P^T chunk by chunk; the weights of 16-key chunk pc + 1 are
      // computed between the MFMAs of chunk pc (half a chunk per step) so this
      // wave's VALU work overlaps its own MFMAs; each step's V^T fragment is
      // read one step ahead.  Same operations and order per value as below.
      static_assert(NDT == 2, "two O^T tiles per chunk");
      float e8[QT][8];
      Frag<T> a = col_v(0, 0);
#pragma unroll
      for (int pc = 0; pc < NPC; ++pc) {
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          const bool last = dt + 1 == NDT;
          Frag<T> a_n = a;
          if (!last || pc + 1 < NPC) a_n = col_v(last ? pc + 1 : pc, last ? 0 : dt + 1);
#pragma unroll
          for (int t = 0; t < QT; ++t) acc[t][dt] = mma(a, pf[t][pc], acc[t][dt]);
          if (pc + 1 < NPC) {
            const int nc = pc + 1;
#pragma unroll
            for (int t = 0; t < QT; ++t)
#pragma unroll
              for (int e = 4 * dt; e < 4 * dt + 4; ++e)
                e8[t][e] = fast_exp2(fmaf(s[nc >> 1][t][8 * (nc & 1) + e], cl2, neg[t]));
          }
          a = a_n;
          __builtin_amdgcn_sched_barrier(0);
        }
        if (pc + 1 < NPC) {
#pragma unroll
          for (int t = 0; t < QT; ++t) {
            pf[t][pc + 1] = to_frag<T>(e8[t]);
            l_run[t] = tree_sum<8>(e8[t], l_run[t]);
          }
        }
      }
      return;
    }
    // O^T += V^T P^T; each V^T fragment feeds every query sub-tile.
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
#pragma unroll
      for (int pc = 0; pc < NPC; ++pc) {
        const Frag<T> a = col_v(pc, dt);
#pragma unroll
        for (int t = 0; t < QT; ++t) acc[t][dt] = mma(a, pf[t][pc], acc[t][dt]);
      }
    }
  };

  // Double-buffered pipeline: the next tile is fetched into registers while
  // the current one is computed, then written to the other LDS stage.  Masked
  // tiles (ragged tail, causal diagonal) run in a separate second loop.
  auto step = [&](auto mask_tag, int it) {
    const bool has_next = it + 1 < n_tiles;
    if (has_next) load_stage(kb + (int64_t)(it + 1) * BK);
    tile(mask_tag, it);
    if (has_next) store_stage((it + 1) & 1);
    __syncthreads();
  };
  if (n_tiles > 0) {
    load_stage(kb);
    store_stage(0);
  }
  __syncthreads();
  int it = 0;
  for (; it < n_plain; ++it) step(BoolC<false>{}, it);
  for (; it < n_tiles; ++it) step(BoolC<true>{}, it);

  // ---- epilogue.
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const float l_tot = xhalf_sum(l_run[t]);
    const int64_t row = qw + 32 * t + c;
    if (row >= p.n_q) continue;
    if (p.n_splits == 1) {
      // A row with no visible key (key padding) has l = 0: o = 0, lse = -inf.
      const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;
      TO* og = static_cast<TO*>(p.o) + head_base(p.so, bh, p.heads) + row * p.so.r;
      TO* gl = p.o_lo ? static_cast<TO*>(p.o_lo) + ((size_t)bh * p.n_q + row) * DV : nullptr;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int a4 = 0; a4 < 4; ++a4) {
          float x4[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) x4[e] = acc[t][dt][4 * a4 + e] * inv;
          const int f = 32 * dt + 8 * a4 + 4 * h;
          store_out4<TO>(og + f, gl ? gl + f : nullptr, x4);
        }
      if (h == 0 && p.lse)
        p.lse[(size_t)bh * p.n_q + row] = l_tot > 0.0f ? (m_ref[t] + __log2f(l_tot)) * kLn2 : -INFINITY;
    } else {
      const size_t prow = ((size_t)split * p.bh + bh) * p.n_q + row;
      float* po = p.part_o + prow * DV;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int a4 = 0; a4 < 4; ++a4) {
          f32x4 v4;
#pragma unroll
          for (int e = 0; e < 4; ++e) v4[e] = acc[t][dt][4 * a4 + e];
          *reinterpret_cast<f32x4*>(po + 32 * dt + 8 * a4 + 4 * h) = v4;
        }
      if (h == 0) {
        p.part_m[prow] = m_ref[t];  // log2 units (scaled), -inf if no visible key
        p.part_l[prow] = l_tot;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Forward for 16-bit inputs (d = 64 and d = 128): two wave groups in opposite
// phases.
//
// A workgroup is 8 waves; wave w and wave w + 4 share a SIMD.  Waves 0-3
// (group 0) and 4-7 (group 1) alternate between an MFMA phase (scores of key
// tile j and the PV product of tile j-1) and a vector phase (the lazy softmax
// of the tile whose scores they computed), one barrier between phases, so that
// on every SIMD one wave feeds the matrix cores while the other runs the
// exponentials.  Group 1 runs one phase behind group 0.  A wave owns 64
// queries at d = 64 and 32 at d = 128 (the registers of the accumulator and
// the query fragments); both give 32 MFMAs per 64-key tile and wave.  K and V tiles go from
// memory to LDS with global_load_lds (no staging registers), issued by group 1
// during its vector phase two phases before they are read; rows are stored
// unpadded with an XOR swizzle of their 16-byte chunks that keeps both the
// row-fragment reads of K and the transposing reads of V free of bank
// conflicts.
// ---------------------------------------------------------------------------
#ifndef MEA_FWD_PP_LEAN_COPY
#define MEA_FWD_PP_LEAN_COPY 1
#endif
#ifndef MEA_FWD_PP_W0
#define MEA_FWD_PP_W0 3
#endif
#ifndef MEA_FWD_PP128_W0
#define MEA_FWD_PP128_W0 0
#endif
// LDS fetch distance (steps) of the d = 128 MFMA phase.
#ifndef MEA_FWD_PP128_AHEAD
#define MEA_FWD_PP128_AHEAD 3
#endif
namespace pp {
// Tile geometry per head dimension.  K and V rows are stored unpadded; the
// physical 16-byte chunk of logical chunk x in row r is x ^ swz(r).
//   d = 64: 128-byte rows, two per 64-bank line.  K is read 16 rows x one
//   chunk per 16 lanes (perm32 rows 0-15): rows 2m, 2m+1 sit in different bank
//   halves and (r >> 1) & 7 spreads the 8 pairs over the 8 chunks.  V is read
//   by the transposing read, 4 rows x 4 chunks per 32 lanes: rows 4m+2, 4m+3
//   move to the other 4 chunks of their half.
//   d = 128: 256-byte rows, one per 64-bank line.  K: r & 15 gives the 16 rows
//   16 different chunks; V: (r & 3) << 2 gives each of the 4 rows its own
//   4-chunk group.
template <int D> struct Cfg;
template <> struct Cfg<64> {
  static constexpr int QT = 2, W0 = MEA_FWD_PP_W0;
  __device__ static __forceinline__ int swz_k(int r) { return (r >> 1) & 7; }
  __device__ static __forceinline__ int swz_v(int r) { return ((r >> 1) & 1) << 2; }
};
template <> struct Cfg<128> {
  static constexpr int QT = 1, W0 = MEA_FWD_PP128_W0;
  __device__ static __forceinline__ int swz_k(int r) { return r & 15; }
  __device__ static __forceinline__ int swz_v(int r) { return (r & 3) << 2; }
};
// Four K/V stages at d = 128 (128 KiB of LDS) measured 0.2-1.6 % faster than
// three (causal 4x32x8192: 2.028 -> 1.995 ms); at d = 64 four were slower.
#ifndef MEA_FWD_PP128_NSTAGE
#define MEA_FWD_PP128_NSTAGE 4
#endif
constexpr int BK = 64, NW = 8;
// K and V stages each: tile j of K lives in stage j % NSTAGE, of V too.
template <int D> constexpr int NSTAGE = D == 128 ? MEA_FWD_PP128_NSTAGE : 3;
template <int D> constexpr int BQ = NW * Cfg<D>::QT * 32;  // queries per workgroup
}  // namespace pp

template <typename T, typename TO, int D, bool CAUSAL>
__global__ __launch_bounds__(512, 1) void attn_fwd_pp_kernel(FwdParams p) {
  using pp::BK;
  constexpr int NSTAGE = pp::NSTAGE<D>;
  using pp::NW;
  using C = pp::Cfg<D>;
  constexpr int QT = C::QT, BQ = pp::BQ<D>;
  constexpr int ROWB = D * 2;              // bytes per LDS row (unpadded)
  constexpr int TILEB = BK * ROWB;         // one K or V tile: 8 or 16 KiB
  constexpr int CPR = ROWB / 16;           // 16-byte chunks per row
  constexpr int RPU = 1024 / ROWB;         // rows per 1 KiB copy instruction
  constexpr int UPW = TILEB / 1024 / 4;    // copy instructions per group-1 wave and tile
  constexpr int KC = D / 16, NKT = BK / 32, NPC = BK / 16, NDT = D / 32;
  auto swz_k = [](int r) { return C::swz_k(r); };
  auto swz_v = [](int r) { return C::swz_v(r); };
  // 16-key chunks of query sub-tile 0 whose weights are computed in the MFMA
  // phase (interleaved with the PV MFMAs); the rest go to the softmax phase.
  constexpr int W0 = C::W0;
  static_assert(W0 >= 0 && W0 <= NPC, "weight chunks");
  static_assert(sizeof(T) == 2, "16-bit inputs only");

  // NSTAGE stages each of K and V: tile j of K lives in kst[j % NSTAGE], of V
  // in vst[j % NSTAGE].
  __shared__ __align__(16) unsigned char kst[NSTAGE * TILEB], vst[NSTAGE * TILEB];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int grp = wave >> 2;
  const int lane = tid & 63;
  const int h = lane >> 5, c = lane & 31;

  const int w = xcd_remap(blockIdx.x, gridDim.x);
  const int qt_idx = w % p.n_qtiles;
  const int rest = w / p.n_qtiles;
  const int bh = bh_of_group(rest % p.bh, p.bh, p.heads);
  const int split = rest / p.bh;
  const int qtile = CAUSAL ? (p.n_qtiles - 1 - qt_idx) : qt_idx;
  const int64_t q0 = (int64_t)qtile * BQ;
  const int64_t qw = q0 + (int64_t)wave * QT * 32;

  const T* __restrict__ qg = static_cast<const T*>(p.q) + head_base(p.sq, bh, p.heads);
  const T* __restrict__ kg = static_cast<const T*>(p.k) + head_base(p.sk, bh, p.heads);
  const T* __restrict__ vg = static_cast<const T*>(p.v) + head_base(p.sv, bh, p.heads);

  // Keys visible to this (batch, head): n_k, or the batch's valid length
  // (key padding); loads stay bounded by n_k.
  const int64_t n_k = valid_keys(p.kv_len, bh, p.heads, p.n_k);
  const int64_t kb = (int64_t)split * p.keys_per_split;
  int64_t ke = kb + p.keys_per_split;
  if (ke > n_k) ke = n_k;
  if (CAUSAL && ke > q0 + BQ) ke = q0 + BQ;
  const int n_tiles = ke > kb ? (int)((ke - kb + BK - 1) / BK) : 0;
  int n_plain = n_tiles;
  {
    const int64_t full = n_k > kb ? (n_k - kb) / BK : 0;
    if (full < n_plain) n_plain = (int)full;
    if (CAUSAL) {
      const int64_t below = q0 - kb + 1 > 0 ? (q0 - kb + 1) / BK : 0;
      if (below < n_plain) n_plain = (int)below;
    }
  }

  Frag<T> qf[QT][KC];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const int64_t row = qw + 32 * t + c;
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
      if (row < p.n_q) {
        qf[t][kc] = *reinterpret_cast<const Frag<T>*>(qg + row * p.sq.r + 16 * kc + 8 * h);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[t][kc][e] = (T)0.0f;
      }
    }
  }
  wait_global_loads();

  f32x16 acc[QT][NDT];
#pragma unroll
  for (int t = 0; t < QT; ++t)
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[t][dt][r] = 0.0f;
  float m_ref[QT], l_run[QT];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    m_ref[t] = -INFINITY;
    l_run[t] = 0.0f;
  }
  const float cl2 = p.scale_log2;

  auto kstage = [&](int j) { return kst + (j % NSTAGE) * TILEB; };
  auto vstage = [&](int j) { return vst + (j % NSTAGE) * TILEB; };

  // Asynchronous copy of rows [k0, k0 + BK) of K or V into an LDS stage.  One
  // instruction moves 1 KiB = RPU rows; the lane writing physical chunk x of
  // row r fetches logical chunk x ^ swz(r).  Rows past n_k repeat the last key
  // row (finite data; those keys are masked).
  auto load_tile = [&](const T* g, int64_t k0, unsigned char* stage, bool is_v, int part, int nparts)
                       __attribute__((always_inline)) {
    const int64_t rs = is_v ? p.sv.r : p.sk.r;
    for (int ii = part; ii < BK / RPU; ii += nparts) {
      const int row = RPU * ii + (int)((unsigned)lane / CPR);
      const int x = (int)((unsigned)lane % CPR);
      const int lchunk = x ^ (is_v ? swz_v(row) : swz_k(row));
      int64_t key = k0 + row;
      if (key > p.n_k - 1) key = p.n_k - 1;
      const T* src = g + key * rs + lchunk * 8;
      copy_to_lds16(src, __builtin_amdgcn_readfirstlane(lds_addr(stage) + ii * 1024));
    }
  };

  // S^T of tile j for both query sub-tiles.
  auto scores = [&](const unsigned char* ks, f32x16 (&s)[NKT][QT]) __attribute__((always_inline)) {
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int t = 0; t < QT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[kt][t][r] = 0.0f;
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        const int row = 32 * kt + perm32(c);
        const int x = (2 * kc + h) ^ swz_k(row);
        const Frag<T> a = *reinterpret_cast<const Frag<T>*>(ks + row * ROWB + x * 16);
#pragma unroll
        for (int t = 0; t < QT; ++t) s[kt][t] = mma(a, qf[t][kc], s[kt][t]);
      }
    }
  };

  // O^T += V^T P^T for tile j: the V^T column fragments come from the
  // transposing LDS read (see lds_col_frag), with the V swizzle applied.
  auto pv = [&](const unsigned char* vs, Frag<T> (&pf)[QT][NPC]) __attribute__((always_inline)) {
    const int g = lane >> 4, i = lane & 15;
    // One sub-tile (d = 128): feature tiles vary fastest, so consecutive MFMAs
    // accumulate into different registers.
    constexpr int NA = QT == 1 ? NPC : NDT, NB = QT == 1 ? NDT : NPC;
#pragma unroll
    for (int ia = 0; ia < NA; ++ia) {
#pragma unroll
      for (int ib = 0; ib < NB; ++ib) {
        const int dt = QT == 1 ? ib : ia, pc = QT == 1 ? ia : ib;
        const int row = 16 * pc + 8 * (g >> 1) + (i >> 2);
        const int colb = 2 * (32 * dt + 16 * (g & 1) + 4 * (i & 3));
        const int addr_lo = row * ROWB + (((colb >> 4) ^ swz_v(row)) << 4) + (colb & 15);
        const int addr_hi = (row + 4) * ROWB + (((colb >> 4) ^ swz_v(row + 4)) << 4) + (colb & 15);
        const v4s_t lo = lds_read_tr16(vs + addr_lo);
        const v4s_t hi = lds_read_tr16(vs + addr_hi);
        typedef short v8s_t __attribute__((ext_vector_type(8)));
        v8s_t r8;
        r8[0] = lo[0]; r8[1] = lo[1]; r8[2] = lo[2]; r8[3] = lo[3];
        r8[4] = hi[0]; r8[5] = hi[1]; r8[6] = hi[2]; r8[7] = hi[3];
        const Frag<T> a = __builtin_bit_cast(Frag<T>, r8);
#pragma unroll
        for (int t = 0; t < QT; ++t) acc[t][dt] = mma(a, pf[t][pc], acc[t][dt]);
      }
    }
  };
  (void)pv;

  // Lazy softmax (Section 3) of query sub-tile t of tile j: P = 2^(c s - m)
  // against the current reference m, rounded into pfo[t], and the lane's
  // partial row sum added to l.  The reference has to rise only when a weight
  // would exceed 2^kRescaleSlack; a lane sum above that bound (or not finite,
  // or no reference yet) flags it, and the flagged sub-tile is redone against
  // the tile's true maximum, rescaling the running numerator and denominator.
  // The common path thus needs no row maximum at all.
  auto mask_sub = [&](int j, auto t_tag, f32x16 (&s)[NKT][QT]) __attribute__((always_inline)) {
    constexpr int t = decltype(t_tag)::value;
    const int64_t k0 = kb + (int64_t)j * BK;
    const int key_lim = (int)(n_k - k0 < BK ? n_k - k0 : BK);
    const int lim_c = CAUSAL ? (int)(qw - k0) + c + 32 * t + 1 : BK;
    const int lim = lim_c < key_lim ? lim_c : key_lim;
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (32 * kt + permuted_row(r, h) >= lim) s[kt][t][r] = -INFINITY;
  };
  auto weights = [&](auto t_tag, f32x16 (&s)[NKT][QT], Frag<T> (&pfo)[QT][NPC], float neg, int pc0 = 0)
                     __attribute__((always_inline)) {
    constexpr int t = decltype(t_tag)::value;
    float sum0 = 0.0f, sum1 = 0.0f;
#pragma unroll
    for (int pc = pc0; pc < NPC; ++pc) {
      float e8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) e8[e] = fast_exp2(fmaf(s[pc >> 1][t][8 * (pc & 1) + e], cl2, neg));
      pfo[t][pc] = to_frag<T>(e8);
      if (pc & 1) sum1 = tree_sum<8>(e8, sum1);
      else sum0 = tree_sum<8>(e8, sum0);
    }
    return sum0 + sum1;
  };
  auto finish_sub = [&](auto t_tag, f32x16 (&s)[NKT][QT], Frag<T> (&pfo)[QT][NPC], float tsum)
                        __attribute__((always_inline)) {
    constexpr int t = decltype(t_tag)::value;
    const bool redo = !(tsum <= kRescaleBound) || m_ref[t] == -INFINITY;
    if (__builtin_amdgcn_ballot_w64(redo)) {
      // Rare path: keep it a branch (an empty volatile statement cannot be
      // speculated, so the compiler does not flatten it into the common path).
      asm volatile("");
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kt][t][r]);
      const float m_new = fmaxf(m_ref[t], xhalf_max(mx) * cl2);
      const float alpha = m_new == -INFINITY ? 1.0f : fast_exp2(m_ref[t] - m_new);
      l_run[t] *= alpha;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[t][dt][r] *= alpha;
      m_ref[t] = m_new;
      tsum = weights(t_tag, s, pfo, m_new == -INFINITY ? 0.0f : -m_new);
    }
    l_run[t] += tsum;
  };
  // O += V(j-1) P(j-1) for both sub-tiles, interleaved step by step with the
  // weights of sub-tile 0 of tile j (a wave issues VALU work slowly, so it
  // fills the gaps between its own MFMAs).  Returns that sub-tile's lane sum.
  auto pv_weights0 = [&](const unsigned char* vs, Frag<T> (&pf_old)[QT][NPC], Frag<T> (&pf_new)[QT][NPC],
                         f32x16 (&s)[NKT][QT], float neg) __attribute__((always_inline)) {
    constexpr int NSTEP = NDT * NPC;
    // With one query sub-tile per wave (d = 128) consecutive steps go to
    // different accumulators (the feature tile varies fastest), so no MFMA
    // waits for the result of the one before it, and the V fragments are
    // read two steps ahead (one step is a single 32-cycle MFMA there).
    constexpr bool DT_FAST = QT == 1;
    constexpr int AHEAD = QT == 1 ? 2 : 1;
    const int g = lane >> 4, i4 = lane & 15;
    auto vfrag = [&](int step) __attribute__((always_inline)) {
      const int dt = DT_FAST ? step % NDT : step / NPC, pc = DT_FAST ? step / NDT : step % NPC;
      const int row = 16 * pc + 8 * (g >> 1) + (i4 >> 2);
      const int colb = 2 * (32 * dt + 16 * (g & 1) + 4 * (i4 & 3));
      const int addr_lo = row * ROWB + (((colb >> 4) ^ swz_v(row)) << 4) + (colb & 15);
      const int addr_hi = (row + 4) * ROWB + (((colb >> 4) ^ swz_v(row + 4)) << 4) + (colb & 15);
      const v4s_t lo = lds_read_tr16(vs + addr_lo);
      const v4s_t hi = lds_read_tr16(vs + addr_hi);
      typedef short v8s_t __attribute__((ext_vector_type(8)));
      v8s_t r8;
      r8[0] = lo[0]; r8[1] = lo[1]; r8[2] = lo[2]; r8[3] = lo[3];
      r8[4] = hi[0]; r8[5] = hi[1]; r8[6] = hi[2]; r8[7] = hi[3];
      return __builtin_bit_cast(Frag<T>, r8);
    };
    Frag<T> vf[AHEAD + 1];
    vf[0] = vfrag(0);
    if constexpr (AHEAD > 1) vf[1] = vfrag(1);
    u32x4 packed;
    float sum0 = 0.0f, sum1 = 0.0f;
#pragma unroll
    for (int i = 0; i < NSTEP; ++i) {
      const int dt = DT_FAST ? i % NDT : i / NPC, pcv = DT_FAST ? i / NDT : i % NPC;
      if constexpr (AHEAD == 1) {
        if (i + 1 < NSTEP) vf[(i + 1) & 1] = vfrag(i + 1);
      } else {
        if (i + AHEAD < NSTEP) vf[(i + AHEAD) % (AHEAD + 1)] = vfrag(i + AHEAD);
      }
      // Step i does half of chunk pcs of the weights; with W0 < NPC chunks
      // here, the steps are spread evenly over the PV MFMAs.
      constexpr int WSTEPS = 2 * W0;
      const int wi = (i * WSTEPS) / NSTEP;
      const bool has_w = WSTEPS > 0 && (i * WSTEPS) % NSTEP < WSTEPS;
      const int pcs = wi >> 1, half = wi & 1;
      acc[0][dt] = mma(vf[AHEAD == 1 ? (i & 1) : i % (AHEAD + 1)], pf_old[0][pcv], acc[0][dt]);
      if (has_w) {
        float e4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          e4[e] = fast_exp2(fmaf(s[pcs >> 1][0][8 * (pcs & 1) + 4 * half + e], cl2, neg));
        packed[2 * half] = pack2<T>(e4[0], e4[1]);
        packed[2 * half + 1] = pack2<T>(e4[2], e4[3]);
        if (pcs & 1) sum1 = tree_sum<4>(e4, sum1);
        else sum0 = tree_sum<4>(e4, sum0);
      }
#pragma unroll
      for (int t = 1; t < QT; ++t) acc[t][dt] = mma(vf[AHEAD == 1 ? (i & 1) : i % (AHEAD + 1)], pf_old[t][pcv], acc[t][dt]);
      if (has_w && half) pf_new[0][pcs] = __builtin_bit_cast(Frag<T>, packed);
      __builtin_amdgcn_sched_barrier(0);
    }
    return sum0 + sum1;
  };
  // The copies into LDS are invisible to the compiler (inline assembly), so
  // the barrier also fences the compiler: no LDS access moves across it.
  auto barrier = [&]() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" ::: "memory");
  };

  // Every wave runs the same sequence -- MFMA phase of tile j, barrier,
  // softmax phase of tile j, barrier -- and group 1 starts one barrier later,
  // so its MFMA phases coincide with group 0's softmax phases.  A wave issues
  // at most about one VALU instruction per 7 cycles, so the softmax is split:
  // sub-tile 0 is computed in the MFMA phase, interleaved with O += V P of the
  // previous tile, and sub-tile 1 in the softmax phase.  Group 1 also moves the
  // tiles: in its softmax phase of tile j it issues K(j+3) (into the stage of
  // K(j+3-NSTAGE)) and V(j+2) (into the stage of V(j+2-NSTAGE)); with three
  // stages those are K(j) and V(j-1), last read in global phases 2j and
  // 2j+1, and with four an older tile each.  Before the barrier that ends its
  // MFMA phase of tile j it waits for K(j+1) and V(j), issued two softmax
  // phases earlier, letting the copies of the last softmax phase run on.
  f32x16 s[NKT][QT];
  Frag<T> pfa[QT][NPC], pfb[QT][NPC];
#pragma unroll
  for (int t = 0; t < QT; ++t)
#pragma unroll
    for (int pc = 0; pc < NPC; ++pc)
#pragma unroll
      for (int e = 0; e < 8; ++e) pfb[t][pc][e] = (T)0.0f;
  // Tile 0 multiplies the V(-1) stage by zero weights: clear it so that it
  // holds finite values.
  reinterpret_cast<u32x4*>(vstage(NSTAGE - 1))[tid] = u32x4{0u, 0u, 0u, 0u};
  if constexpr (TILEB > NW * 64 * 16)
    reinterpret_cast<u32x4*>(vstage(NSTAGE - 1))[tid + NW * 64] = u32x4{0u, 0u, 0u, 0u};
  static_assert(TILEB == NW * 64 * 16 || TILEB == 2 * NW * 64 * 16, "one or two 16-byte stores per thread clear a stage");
  if (n_tiles > 0) load_tile(kg, kb, kstage(0), false, wave, NW);  // K(0): 1 KiB per wave and instruction
  // The barrier's fence does not cover copies the compiler cannot see.
  wait_global_loads();
  __syncthreads();
  // Group 1 issues two waves of copies ahead, as if from softmax phases -2
  // and -1, and starts one phase behind group 0.  Its wave w copies units
  // w - 4 + 4i, i < UPW (rows RPU u .. RPU u + RPU - 1) of each tile; the
  // lane's source offsets within a tile (bytes) are computed once.
  constexpr unsigned E = sizeof(T);
  const unsigned rk = (unsigned)p.sk.r, rv = (unsigned)p.sv.r;  // row strides (< 2^24, checked on the host)
  constexpr int LCPR = CPR == 8 ? 3 : 4;
  static_assert(CPR == 1 << LCPR && (UPW == 2 || UPW == 4), "copy geometry");
  const int urow0 = RPU * (wave - 4) + (lane >> LCPR), urow1 = urow0 + 4 * RPU;
  const unsigned uk0 = E * (urow0 * rk + 8 * ((lane & (CPR - 1)) ^ swz_k(urow0)));
  const unsigned uk1 = E * (urow1 * rk + 8 * ((lane & (CPR - 1)) ^ swz_k(urow1)));
  const unsigned uv0 = E * (urow0 * rv + 8 * ((lane & (CPR - 1)) ^ swz_v(urow0)));
  const unsigned uv1 = E * (urow1 * rv + 8 * ((lane & (CPR - 1)) ^ swz_v(urow1)));
  // d = 128: units w - 4 + 8 and w - 4 + 12 as well.
  const int urow2 = urow0 + 8 * RPU, urow3 = urow0 + 12 * RPU;
  const unsigned uk2 = UPW > 2 ? E * (urow2 * rk + 8 * ((lane & (CPR - 1)) ^ swz_k(urow2))) : 0u;
  const unsigned uk3 = UPW > 2 ? E * (urow3 * rk + 8 * ((lane & (CPR - 1)) ^ swz_k(urow3))) : 0u;
  const unsigned uv2 = UPW > 2 ? E * (urow2 * rv + 8 * ((lane & (CPR - 1)) ^ swz_v(urow2))) : 0u;
  const unsigned uv3 = UPW > 2 ? E * (urow3 * rv + 8 * ((lane & (CPR - 1)) ^ swz_v(urow3))) : 0u;
  auto copy_tile = [&](bool is_v, int j, unsigned char* stage, unsigned off0, unsigned off1, unsigned off2,
                       unsigned off3) __attribute__((always_inline)) {
    const int64_t k0 = kb + (int64_t)j * BK;
    const unsigned base = __builtin_amdgcn_readfirstlane(lds_addr(stage) + (wave - 4) * 1024);
    const T* g = is_v ? vg : kg;
    if (k0 + BK <= p.n_k) {
      const T* tile = g + k0 * (is_v ? p.sv.r : p.sk.r);
      copy_to_lds16_sb(tile, off0, base);
      copy_to_lds16_sb(tile, off1, base + 4096);
      if constexpr (UPW > 2) {
        copy_to_lds16_sb(tile, off2, base + 8192);
        copy_to_lds16_sb(tile, off3, base + 12288);
      }
    } else {
      load_tile(g, k0, stage, is_v, wave - 4, 4);
    }
  };
  // LEAN (causal, d = 64): the register allocator spilled the offsets above
  // and reloaded them before each tile's copies, and the reload's wait
  // (vmcnt 0) also waited for the copies still in flight.  Instead the lane
  // offset is recomputed at each issue from an opaque copy of the lane index
  // (a few VALU instructions), one per tensor: the wave's units are 4 RPU
  // rows apart and both swizzles repeat every 16 rows, so the row shift goes
  // into the scalar base.
  constexpr bool LEAN = MEA_FWD_PP_LEAN_COPY && CAUSAL && D == 64;
  static_assert(!LEAN || (4 * RPU) % 16 == 0, "swizzle period");
  auto copy_tile_lean = [&](bool is_v, int j, unsigned char* stage) __attribute__((always_inline)) {
    const int64_t k0 = kb + (int64_t)j * BK;
    const unsigned base = __builtin_amdgcn_readfirstlane(lds_addr(stage) + (wave - 4) * 1024);
    const T* g = is_v ? vg : kg;
    if (k0 + BK <= p.n_k) {
      int l = lane;
      asm volatile("" : "+v"(l));
      const int row = RPU * (wave - 4) + (l >> LCPR);
      const int x = (l & (CPR - 1)) ^ (is_v ? swz_v(row) : swz_k(row));
      const int64_t rs = is_v ? p.sv.r : p.sk.r;
      const unsigned off = E * ((unsigned)row * (unsigned)rs + 8u * (unsigned)x);
      const T* tile = g + k0 * rs;
#pragma unroll
      for (int i = 0; i < UPW; ++i) copy_to_lds16_sb(tile + 4 * RPU * i * rs, off, base + 4096 * i);
    } else {
      load_tile(g, k0, stage, is_v, wave - 4, 4);
    }
  };
  auto issue = [&](int j) __attribute__((always_inline)) {
    if constexpr (LEAN) {
      if (j + 3 < n_tiles) copy_tile_lean(false, j + 3, kstage(j + 3));
      if (j + 2 < n_tiles) copy_tile_lean(true, j + 2, vstage(j + 2));
    } else {
      if (j + 3 < n_tiles) copy_tile(false, j + 3, kstage(j + 3), uk0, uk1, uk2, uk3);
      if (j + 2 < n_tiles) copy_tile(true, j + 2, vstage(j + 2), uv0, uv1, uv2, uv3);
    }
  };
  if (grp == 1) {
    issue(-2);
    issue(-1);
    barrier();
  }
  // pf_old holds P(j-1) and pf_new receives P(j).
  // MFMA phase with one query sub-tile per wave (d = 128): S = K Q^T of tile
  // j and O += V P of tile j - 1 as one sequence of 32 single-MFMA steps, S
  // and PV steps alternating (consecutive MFMAs accumulate into different
  // registers), each step's LDS fragment read PF_AHEAD steps before its MFMA.
  // A lone MFMA does not cover an LDS read's latency, so the fragments of the
  // next steps must already be in flight.
  auto mfma_phase1 = [&](const unsigned char* ks, const unsigned char* vs, Frag<T> (&pf_old)[QT][NPC],
                         f32x16 (&sc)[NKT][QT]) __attribute__((always_inline)) {
    constexpr int NS = KC * NKT, NP = NDT * NPC;
    static_assert(QT != 1 || NS == NP, "alternating S and PV steps");
    constexpr int N = NS + NP, AH = MEA_FWD_PP128_AHEAD;
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) sc[kt][0][r] = 0.0f;
    const int g = lane >> 4, i4 = lane & 15;
    auto frag = [&](int step) __attribute__((always_inline)) {
      const int k = step >> 1;
      if ((step & 1) == 0) {  // S step k: key sub-tile k % NKT, k chunk k / NKT
        const int row = 32 * (k % NKT) + perm32(c);
        const int x = (2 * (k / NKT) + h) ^ swz_k(row);
        return *reinterpret_cast<const Frag<T>*>(ks + row * ROWB + x * 16);
      }
      const int dt = k % NDT, pc = k / NDT;  // PV step k
      const int row = 16 * pc + 8 * (g >> 1) + (i4 >> 2);
      const int colb = 2 * (32 * dt + 16 * (g & 1) + 4 * (i4 & 3));
      const int addr_lo = row * ROWB + (((colb >> 4) ^ swz_v(row)) << 4) + (colb & 15);
      const int addr_hi = (row + 4) * ROWB + (((colb >> 4) ^ swz_v(row + 4)) << 4) + (colb & 15);
      const v4s_t lo = lds_read_tr16(vs + addr_lo);
      const v4s_t hi = lds_read_tr16(vs + addr_hi);
      typedef short v8s_t __attribute__((ext_vector_type(8)));
      v8s_t r8;
      r8[0] = lo[0]; r8[1] = lo[1]; r8[2] = lo[2]; r8[3] = lo[3];
      r8[4] = hi[0]; r8[5] = hi[1]; r8[6] = hi[2]; r8[7] = hi[3];
      return __builtin_bit_cast(Frag<T>, r8);
    };
    Frag<T> ring[AH + 1];
#pragma unroll
    for (int a = 0; a < AH; ++a) ring[a] = frag(a);
#pragma unroll
    for (int i = 0; i < N; ++i) {
      if (i + AH < N) ring[(i + AH) % (AH + 1)] = frag(i + AH);
      const int k = i >> 1;
      if ((i & 1) == 0) sc[k % NKT][0] = mma(ring[i % (AH + 1)], qf[0][k / NKT], sc[k % NKT][0]);
      else acc[0][k % NDT] = mma(ring[i % (AH + 1)], pf_old[0][k / NDT], acc[0][k % NDT]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  auto iteration = [&](auto mask_tag, int j, Frag<T> (&pf_old)[QT][NPC], Frag<T> (&pf_new)[QT][NPC])
                       __attribute__((always_inline)) {
    const unsigned char* kcur = kstage(j);
    const unsigned char* vprev = vstage(j + NSTAGE - 1);
    constexpr bool MASK = decltype(mask_tag)::value;
    mfma_phase_priority();
    float tsum0 = 0.0f;
    if constexpr (QT == 1 && W0 == 0) {
      mfma_phase1(kcur, vprev, pf_old, s);
    } else {
      scores(kcur, s);
      if constexpr (MASK) mask_sub(j, IntC<0>{}, s);
      tsum0 = pv_weights0(vprev, pf_old, pf_new, s, -m_ref[0]);
      if constexpr (W0 == NPC) finish_sub(IntC<0>{}, s, pf_new, tsum0);
    }
    // Only group 1 has copies in flight (UPW per wave, tile and tensor); the
    // wait is a no-op for group 0.
    if (j + 2 < n_tiles) wait_global_loads_upto<2 * UPW>();
    else if (j + 1 < n_tiles) wait_global_loads_upto<UPW>();
    else wait_global_loads();
    barrier();
    valu_phase_priority();
    if constexpr (QT == 1 && W0 == 0 && MASK) mask_sub(j, IntC<0>{}, s);
    if constexpr (W0 < NPC) finish_sub(IntC<0>{}, s, pf_new, tsum0 + weights(IntC<0>{}, s, pf_new, -m_ref[0], W0));
    if constexpr (QT == 2) {
      if constexpr (MASK) mask_sub(j, IntC<QT - 1>{}, s);
      finish_sub(IntC<QT - 1>{}, s, pf_new, weights(IntC<QT - 1>{}, s, pf_new, -m_ref[QT - 1]));
    }
    if (grp == 1) issue(j);
    barrier();
  };
  auto copy_p = [&](Frag<T> (&dst)[QT][NPC], const Frag<T> (&src)[QT][NPC]) __attribute__((always_inline)) {
#pragma unroll
    for (int t = 0; t < QT; ++t)
#pragma unroll
      for (int pc = 0; pc < NPC; ++pc) dst[t][pc] = src[t][pc];
  };
  // Plain tiles and masked tiles (ragged tail, causal diagonal) run in
  // separate loops; a per-tile branch between the two softmax variants would
  // keep both variants' registers live.  The plain loop is unrolled by two so
  // that the weight buffers it touches are known at compile time.
  int j = 0;
  for (; j + 2 <= n_plain; j += 2) {
    iteration(BoolC<false>{}, j, pfb, pfa);
    iteration(BoolC<false>{}, j + 1, pfa, pfb);
  }
  // Here and after every later tile, pfb holds the weights of tile j - 1.
  if (j < n_plain) {
    iteration(BoolC<false>{}, j, pfb, pfa);
    copy_p(pfb, pfa);
    ++j;
  }
  for (; j < n_tiles; ++j) {
    iteration(BoolC<true>{}, j, pfb, pfa);
    copy_p(pfb, pfa);
  }
  if (n_tiles > 0) pv(vstage(n_tiles - 1), pfb);
  barrier();
  barrier();
  if (grp == 0) barrier();  // same number of barriers in both groups

#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const float l_tot = xhalf_sum(l_run[t]);
    const int64_t row = qw + 32 * t + c;
    if (row >= p.n_q) continue;
    if (p.n_splits == 1) {
      // A row with no visible key (key padding) has l = 0: o = 0, lse = -inf.
      const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;
      TO* og = static_cast<TO*>(p.o) + head_base(p.so, bh, p.heads) + row * p.so.r;
      TO* gl = p.o_lo ? static_cast<TO*>(p.o_lo) + ((size_t)bh * p.n_q + row) * D : nullptr;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int a4 = 0; a4 < 4; ++a4) {
          float x4[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) x4[e] = acc[t][dt][4 * a4 + e] * inv;
          const int f = 32 * dt + 8 * a4 + 4 * h;
          store_out4<TO>(og + f, gl ? gl + f : nullptr, x4);
        }
      if (h == 0 && p.lse)
        p.lse[(size_t)bh * p.n_q + row] = l_tot > 0.0f ? (m_ref[t] + __log2f(l_tot)) * kLn2 : -INFINITY;
    } else {
      const size_t prow = ((size_t)split * p.bh + bh) * p.n_q + row;
      float* po = p.part_o + prow * D;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int a4 = 0; a4 < 4; ++a4) {
          f32x4 v4;
#pragma unroll
          for (int e = 0; e < 4; ++e) v4[e] = acc[t][dt][4 * a4 + e];
          *reinterpret_cast<f32x4*>(po + 32 * dt + 8 * a4 + 4 * h) = v4;
        }
      if (h == 0) {
        p.part_m[prow] = m_ref[t];
        p.part_l[prow] = l_tot;
      }
    }
  }
}

// Combine of the per-split summaries (Section 4): global max, rescale each
// split's numerator and denominator by e^{m_s - m_g}, add, divide.  One thread
// per (row, 4 features).
template <typename TO, int D>
__global__ __launch_bounds__(256) void attn_combine_kernel(FwdParams p) {
  constexpr int G = D / 4;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t rows = (int64_t)p.bh * p.n_q;
  if (gid >= rows * G) return;
  const int64_t row = gid / G;
  const int f0 = 4 * (int)(gid % G);
  const size_t stride = (size_t)rows;
  // At most kCombineGroup summaries reach this kernel (launch_combine stages
  // larger counts), so every load is issued up front: two dependent rounds of
  // loads instead of one per summary.
  constexpr int NS = kCombineGroup;
  const int n = p.n_splits;
  float ms[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) ms[s] = s < n ? p.part_m[s * stride + row] : -INFINITY;
  float m_g = -INFINITY;
#pragma unroll
  for (int s = 0; s < NS; ++s) m_g = fmaxf(m_g, ms[s]);
  float l = 0.0f;
  f32x4 o = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    if (s < n) {
      const float wgt = ms[s] == -INFINITY ? 0.0f : fast_exp2(ms[s] - m_g);
      l += wgt * p.part_l[s * stride + row];
      const f32x4 ps = *reinterpret_cast<const f32x4*>(p.part_o + (s * stride + row) * D + f0);
      o += wgt * ps;
    }
  }
  // No visible key in any range (key padding): o = 0, lse = -inf.
  const float inv = l > 0.0f ? 1.0f / l : 0.0f;
  float x4[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) x4[e] = o[e] * inv;
  const int bh = (int)(row / p.n_q);
  TO* og = static_cast<TO*>(p.o) + head_base(p.so, bh, p.heads) + (row - (int64_t)bh * p.n_q) * p.so.r;
  TO* gl = p.o_lo ? static_cast<TO*>(p.o_lo) + row * D : nullptr;
  store_out4<TO>(og + f0, gl ? gl + f0 : nullptr, x4);
  if (f0 == 0 && p.lse) p.lse[row] = l > 0.0f ? (m_g + __log2f(l)) * kLn2 : -INFINITY;
}

// One stage of the combine: each output range g summarises input ranges
// g G .. g G + G - 1 (fewer at the end) of the same row: maximum m_g, and the
// numerator and denominator rescaled by 2^(m_s - m_g) and added -- the same
// algebra as the final combine, without the division.  One thread per
// (row, output range, 4 features); the G inputs are read together.
template <int D>
__global__ __launch_bounds__(256) void attn_combine_stage_kernel(const float* __restrict__ po,
                                                                 const float* __restrict__ pm,
                                                                 const float* __restrict__ pl, int s_in,
                                                                 float* __restrict__ qo, float* __restrict__ qm,
                                                                 float* __restrict__ ql, int s_out, int64_t rows) {
  constexpr int G4 = D / 4;
  constexpr int G = kCombineGroup;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= rows * s_out * G4) return;
  const int64_t row = gid / ((int64_t)s_out * G4);
  const int rem = (int)(gid % ((int64_t)s_out * G4));
  const int g = rem / G4, f0 = 4 * (rem % G4);
  const int s0 = g * G;
  const int n = s_in - s0 < G ? s_in - s0 : G;
  float ms[G];
#pragma unroll
  for (int i = 0; i < G; ++i) ms[i] = i < n ? pm[(size_t)(s0 + i) * rows + row] : -INFINITY;
  float m_g = -INFINITY;
#pragma unroll
  for (int i = 0; i < G; ++i) m_g = fmaxf(m_g, ms[i]);
  float l = 0.0f;
  f32x4 o = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int i = 0; i < G; ++i) {
    if (i < n) {
      const size_t prow = (size_t)(s0 + i) * rows + row;
      const float wgt = ms[i] == -INFINITY ? 0.0f : fast_exp2(ms[i] - m_g);
      l += wgt * pl[prow];
      o += wgt * *reinterpret_cast<const f32x4*>(po + prow * D + f0);
    }
  }
  const size_t orow = (size_t)g * rows + row;
  *reinterpret_cast<f32x4*>(qo + orow * D + f0) = o;
  if (f0 == 0) {
    qm[orow] = m_g;
    ql[orow] = l;
  }
}

// ---------------------------------------------------------------- launchers

// Combine of the key ranges' summaries into o and lse: stages of
// kCombineGroup ranges while more remain, alternating between the two
// partial buffers, then the final combine.
template <typename TO, int D>
static hipError_t launch_combine(const FwdParams& p, hipStream_t stream) {
  FwdParams pf = p;
  const int64_t rows = (int64_t)p.bh * p.n_q;
  bool in_first = true;
  while (pf.n_splits > kCombineGroup) {
    const int s_out = (pf.n_splits + kCombineGroup - 1) / kCombineGroup;
    float* qo = in_first ? p.part2_o : p.part_o;
    float* qm = in_first ? p.part2_m : p.part_m;
    float* ql = in_first ? p.part2_l : p.part_l;
    const int64_t threads = rows * s_out * (D / 4);
    hipLaunchKernelGGL(attn_combine_stage_kernel<D>, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0,
                       stream, pf.part_o, pf.part_m, pf.part_l, pf.n_splits, qo, qm, ql, s_out, rows);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    pf.part_o = qo;
    pf.part_m = qm;
    pf.part_l = ql;
    pf.n_splits = s_out;
    in_first = !in_first;
  }
  void* args[] = {&pf};
  const int64_t threads = rows * (D / 4);
  return hipLaunchKernel(reinterpret_cast<const void*>(attn_combine_kernel<TO, D>),
                         dim3((unsigned)((threads + 255) / 256)), dim3(256), args, 0, stream);
}

template <typename T, typename TO, int D, int DV, int QT, int BK, int OCC, bool CAUSAL>
static hipError_t launch_fwd_impl(const FwdParams& p, hipStream_t stream) {
  using Cfg = FwdTile<T, D, DV, QT, BK>;
  auto kern = attn_fwd_kernel<T, TO, D, DV, QT, BK, OCC, CAUSAL>;
  // The plan's query tiles must be this kernel's (4 waves x QT x 32 queries).
  if (p.n_qtiles != (p.n_q + 128 * QT - 1) / (128 * QT)) return hipErrorInvalidValue;
  const int64_t grid = (int64_t)p.n_qtiles * p.bh * p.n_splits;
  FwdParams pc = p;
  void* args[] = {&pc};
  hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(kern), dim3((unsigned)grid),
                                 dim3(Cfg::NT), args, Cfg::LDS_BYTES, stream);
  if (e != hipSuccess || p.n_splits == 1) return e;
  return launch_combine<TO, DV>(p, stream);
}

template <typename T, typename TO, int D, bool CAUSAL>
static hipError_t launch_fwd_pp(const FwdParams& p, hipStream_t stream) {
  auto kern = attn_fwd_pp_kernel<T, TO, D, CAUSAL>;
  if (p.n_qtiles != (p.n_q + pp::BQ<D> - 1) / pp::BQ<D>) return hipErrorInvalidValue;
  const int64_t grid = (int64_t)p.n_qtiles * p.bh * p.n_splits;
  FwdParams pc = p;
  void* args[] = {&pc};
  hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(kern), dim3((unsigned)grid),
                                 dim3(pp::NW * 64), args, 0, stream);
  if (e != hipSuccess || p.n_splits == 1) return e;
  return launch_combine<TO, D>(p, stream);
}

template <typename T, typename TO, int D>
static hipError_t launch_fwd_dt(const FwdParams& p, bool causal, hipStream_t stream) {
  if constexpr (sizeof(T) == 2 && FwdShape<T, D>::BQ == pp::BQ<D>) {
    // Short or small problems: the 4-wave kernel with 128-query workgroups
    // (the same choice as the host plan's).
    if constexpr (D == 64) {
      if (fwd64_bq(p.n_q, p.bh, causal) == 128)
        return causal ? launch_fwd_impl<T, TO, 64, 64, 1, FwdShape<T, 64>::BK, MEA_T64_FWD_OCC, true>(p, stream)
                      : launch_fwd_impl<T, TO, 64, 64, 1, FwdShape<T, 64>::BK, MEA_T64_FWD_OCC, false>(p, stream);
    } else {
      using S = FwdShape<T, 128>;
      if (fwd128_bq(p.n_q, causal) == kFwdBq4wave128)
        return causal ? launch_fwd_impl<T, TO, 128, 128, S::QT, S::BK, S::OCC, true>(p, stream)
                      : launch_fwd_impl<T, TO, 128, 128, S::QT, S::BK, S::OCC, false>(p, stream);
    }
    return causal ? launch_fwd_pp<T, TO, D, true>(p, stream) : launch_fwd_pp<T, TO, D, false>(p, stream);
  } else {
    constexpr int QT = FwdShape<T, D>::QT, BK = FwdShape<T, D>::BK, OCC = FwdShape<T, D>::OCC;
    return causal ? launch_fwd_impl<T, TO, D, D, QT, BK, OCC, true>(p, stream)
                  : launch_fwd_impl<T, TO, D, D, QT, BK, OCC, false>(p, stream);
  }
}

// Value head dimension DV != D: the 4-wave kernel with the d = 128 tile shape.
template <typename T, typename TO, int D, int DV>
static hipError_t launch_fwd_dv(const FwdParams& p, bool causal, hipStream_t stream) {
  using S = FwdShape<T, 128>;
  return causal ? launch_fwd_impl<T, TO, D, DV, S::QT, S::BK, S::OCC, true>(p, stream)
                : launch_fwd_impl<T, TO, D, DV, S::QT, S::BK, S::OCC, false>(p, stream);
}
template <typename T, typename TO>
static hipError_t launch_fwd_dv_pair(const FwdParams& p, int d, bool causal, hipStream_t stream) {
  return d == 64 ? launch_fwd_dv<T, TO, 64, 128>(p, causal, stream) : launch_fwd_dv<T, TO, 128, 64>(p, causal, stream);
}

template <typename T, int D>
static hipError_t launch_fwd_out(const FwdParams& p, bool causal, bool out_f32, hipStream_t stream) {
  return out_f32 ? launch_fwd_dt<T, float, D>(p, causal, stream) : launch_fwd_dt<T, T, D>(p, causal, stream);
}

hipError_t launch_fwd(const FwdParams& p, int dtype, int d, int dv, bool causal, bool out_f32,
                      hipStream_t stream) {
  if (dv != d) {
    switch (dtype) {
      case 0: return launch_fwd_dv_pair<float, float>(p, d, causal, stream);
      case 1: return out_f32 ? launch_fwd_dv_pair<_Float16, float>(p, d, causal, stream)
                             : launch_fwd_dv_pair<_Float16, _Float16>(p, d, causal, stream);
      case 2: return out_f32 ? launch_fwd_dv_pair<__bf16, float>(p, d, causal, stream)
                             : launch_fwd_dv_pair<__bf16, __bf16>(p, d, causal, stream);
      default: return hipErrorInvalidValue;
    }
  }
  if (fwd_uses_decode(dtype, d, dv, p.n_q)) {
    const hipError_t e = launch_decode(p, dtype, d, causal, out_f32, stream);
    if (e != hipSuccess || p.n_splits == 1) return e;
    const bool f32 = out_f32;
    if (dtype == 1) {
      if (d == 64) return f32 ? launch_combine<float, 64>(p, stream) : launch_combine<_Float16, 64>(p, stream);
      return f32 ? launch_combine<float, 128>(p, stream) : launch_combine<_Float16, 128>(p, stream);
    }
    if (d == 64) return f32 ? launch_combine<float, 64>(p, stream) : launch_combine<__bf16, 64>(p, stream);
    return f32 ? launch_combine<float, 128>(p, stream) : launch_combine<__bf16, 128>(p, stream);
  }
  switch (dtype * 1000 + d) {
    case 0 * 1000 + 64: return launch_fwd_dt<float, float, 64>(p, causal, stream);
    case 0 * 1000 + 128: return launch_fwd_dt<float, float, 128>(p, causal, stream);
    case 1 * 1000 + 64: return launch_fwd_out<_Float16, 64>(p, causal, out_f32, stream);
    case 1 * 1000 + 128: return launch_fwd_out<_Float16, 128>(p, causal, out_f32, stream);
    case 2 * 1000 + 64: return launch_fwd_out<__bf16, 64>(p, causal, out_f32, stream);
    case 2 * 1000 + 128: return launch_fwd_out<__bf16, 128>(p, causal, out_f32, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace mea
