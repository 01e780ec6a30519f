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

// A tile raises the reference maximum only when one of its scores exceeds it
// by more than this many powers of two (weights then stay <= 2^8).
constexpr float kRescaleSlack = 8.0f;
constexpr float kLn2 = 0.6931471805599453f;

template <bool B> struct BoolC { static constexpr bool value = B; };

template <typename T, int D, int QT, int BK>
struct FwdTile {
  static constexpr int NW = 4;
  static constexpr int NT = NW * 64;
  static constexpr int BQ = NW * QT * 32;
  static constexpr int E = sizeof(T);
  static constexpr int RS = D + 16 / E;          // LDS row stride (elements), 16 B pad
  static constexpr int TILE = BK * RS;           // elements per K or V tile
  static constexpr int CPR = D * E / 16;         // 16-byte chunks per row
  static constexpr int CHUNKS = 2 * BK * CPR;    // K and V chunks per stage
  static constexpr int CPT = CHUNKS / NT;        // chunks per thread per stage
  static constexpr int LDS_BYTES = 2 * 2 * TILE * E;  // double-buffered K and V
  static_assert(CHUNKS % NT == 0, "tile must split evenly over the workgroup");
  static_assert(BK % 32 == 0 && D % 32 == 0, "tile shapes are multiples of 32");
};

template <typename T, typename TO, int D, int QT, int BK, bool CAUSAL>
__global__ __launch_bounds__(256, 2) void attn_fwd_kernel(FwdParams p) {
  using Cfg = FwdTile<T, D, QT, BK>;
  constexpr int RS = Cfg::RS;
  constexpr int KC = D / 16;    // 16-wide k chunks of the QK^T contraction
  constexpr int NKT = BK / 32;  // 32-key sub-tiles per tile
  constexpr int NPC = BK / 16;  // 16-key chunks of the PV contraction
  constexpr int NDT = D / 32;   // 32-row tiles of O^T

  extern __shared__ __align__(16) unsigned char smem_raw[];
  T* smem = reinterpret_cast<T*>(smem_raw);

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int h = lane >> 5, c = lane & 31;

  // ---- workgroup -> (split, bh, query tile); heaviest causal tiles first.
  const int w = xcd_remap(blockIdx.x, gridDim.x);
  const int qt_idx = w % p.n_qtiles;
  const int rest = w / p.n_qtiles;
  const int bh = rest % p.bh;
  const int split = rest / p.bh;
  const int qtile = CAUSAL ? (p.n_qtiles - 1 - qt_idx) : qt_idx;
  const int64_t q0 = (int64_t)qtile * Cfg::BQ;
  const int64_t qw = q0 + (int64_t)wave * QT * 32;  // first query of this wave

  const T* __restrict__ qg = static_cast<const T*>(p.q) + (size_t)bh * p.n_q * D;
  const T* __restrict__ kg = static_cast<const T*>(p.k) + (size_t)bh * p.n_k * D;
  const T* __restrict__ vg = static_cast<const T*>(p.v) + (size_t)bh * p.n_k * D;

  const int64_t kb = (int64_t)split * p.keys_per_split;
  int64_t ke = kb + p.keys_per_split;
  if (ke > p.n_k) ke = p.n_k;
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
        qf[t][kc] = *reinterpret_cast<const Frag<T>*>(qg + row * D + 16 * kc + 8 * h);
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
  auto load_stage = [&](int64_t k0) {
#pragma unroll
    for (int i = 0; i < Cfg::CPT; ++i) {
      const int chunk = tid + i * Cfg::NT;
      const int which = chunk / (BK * Cfg::CPR);  // 0 = K, 1 = V
      const int rem = chunk % (BK * Cfg::CPR);
      const int row = rem / Cfg::CPR, col = rem % Cfg::CPR;
      const int64_t key = k0 + row;
      const T* src = (which ? vg : kg) + key * D + col * (16 / Cfg::E);
      stage[i] = key < p.n_k ? ld16(src) : u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto store_stage = [&](int buf) {
    T* base = smem + buf * 2 * Cfg::TILE;
#pragma unroll
    for (int i = 0; i < Cfg::CPT; ++i) {
      const int chunk = tid + i * Cfg::NT;
      const int which = chunk / (BK * Cfg::CPR);
      const int rem = chunk % (BK * Cfg::CPR);
      const int row = rem / Cfg::CPR, col = rem % Cfg::CPR;
      st16(base + which * Cfg::TILE + row * RS + col * (16 / Cfg::E), stage[i]);
    }
  };

  const int krow = perm32(c);  // key row this lane feeds into the A operand
  const float cl2 = p.scale_log2;

  // Number of leading tiles that need no mask: every key exists (no ragged
  // tail) and, under the causal mask, precedes the workgroup's first query.
  int n_plain = n_tiles;
  {
    const int64_t full = (p.n_k - kb) / BK;
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
    const T* ks = smem + (it & 1) * 2 * Cfg::TILE;
    const T* vs = ks + Cfg::TILE;
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
        const Frag<T> a = lds_frag<T>(ks + (32 * kt + krow) * RS + 16 * kc + 8 * h);
#pragma unroll
        for (int t = 0; t < QT; ++t) s[kt][t] = mma(a, qf[t][kc], s[kt][t]);
      }
    }

    if constexpr (MASK) {
      // Tile-relative 32-bit bounds: key k0 + x is valid iff x < key_lim and,
      // under the causal mask, visible to query qw + 32t + c iff x <= q_rel + 32t.
      const int key_lim = (int)(p.n_k - k0 < BK ? p.n_k - k0 : BK);
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
        const float alpha = fast_exp2(m_ref[t] - m_new);  // 0 on the first raise
        l_run[t] *= alpha;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[t][dt][r] *= alpha;
        m_ref[t] = m_new;
      }
      // A row with no visible key so far keeps m_ref = -inf; offset 0 keeps
      // its (all -inf) exponents at weight 0 instead of NaN.
      const float neg = (MASK && m_ref[t] == -INFINITY) ? 0.0f : -m_ref[t];
#pragma unroll
      for (int pc = 0; pc < NPC; ++pc) {
        float e8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) e8[e] = fast_exp2(fmaf(s[pc >> 1][t][8 * (pc & 1) + e], cl2, neg));
        pf[t][pc] = to_frag<T>(e8);
        l_run[t] = frag_sum(pf[t][pc], e8, l_run[t]);
      }
    }
    // O^T += V^T P^T; each V^T fragment feeds every query sub-tile.
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
#pragma unroll
      for (int pc = 0; pc < NPC; ++pc) {
        Frag<T> a;
        if constexpr (sizeof(T) == 2) {
          a = lds_col_frag<T>(vs, RS, 16 * pc, 32 * dt, lane);
        } else {
          a = lds_col_frag_f32(reinterpret_cast<const float*>(vs), RS, 16 * pc, 32 * dt, lane);
        }
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
      const float inv = 1.0f / l_tot;
      TO* og = static_cast<TO*>(p.o) + ((size_t)bh * p.n_q + row) * D;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int a4 = 0; a4 < 4; ++a4) {
          typename FragT<TO>::half v4;
#pragma unroll
          for (int e = 0; e < 4; ++e) v4[e] = (TO)(acc[t][dt][4 * a4 + e] * inv);
          *reinterpret_cast<typename FragT<TO>::half*>(og + 32 * dt + 8 * a4 + 4 * h) = v4;
        }
      if (h == 0 && p.lse)
        p.lse[(size_t)bh * p.n_q + row] = (m_ref[t] + __log2f(l_tot)) * kLn2;
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
        p.part_m[prow] = m_ref[t];  // log2 units (scaled), -inf if no visible key
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
  float m_g = -INFINITY;
  for (int s = 0; s < p.n_splits; ++s) m_g = fmaxf(m_g, p.part_m[s * stride + row]);
  float l = 0.0f;
  f32x4 o = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int s = 0; s < p.n_splits; ++s) {
    const float ms = p.part_m[s * stride + row];
    const float wgt = ms == -INFINITY ? 0.0f : fast_exp2(ms - m_g);
    l += wgt * p.part_l[s * stride + row];
    const f32x4 ps = *reinterpret_cast<const f32x4*>(p.part_o + (s * stride + row) * D + f0);
    o += wgt * ps;
  }
  const float inv = 1.0f / l;
  typename FragT<TO>::half out;
#pragma unroll
  for (int e = 0; e < 4; ++e) out[e] = (TO)(o[e] * inv);
  *reinterpret_cast<typename FragT<TO>::half*>(static_cast<TO*>(p.o) + row * D + f0) = out;
  if (f0 == 0 && p.lse) p.lse[row] = (m_g + __log2f(l)) * kLn2;
}

// ---------------------------------------------------------------- launchers

template <typename T, typename TO, int D, int QT, int BK, bool CAUSAL>
static hipError_t launch_fwd_impl(const FwdParams& p, hipStream_t stream) {
  using Cfg = FwdTile<T, D, QT, BK>;
  auto kern = attn_fwd_kernel<T, TO, D, QT, BK, CAUSAL>;
  const int64_t grid = (int64_t)p.n_qtiles * p.bh * p.n_splits;
  FwdParams pc = p;
  void* args[] = {&pc};
  hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(kern), dim3((unsigned)grid),
                                 dim3(Cfg::NT), args, Cfg::LDS_BYTES, stream);
  if (e != hipSuccess || p.n_splits == 1) return e;
  auto comb = attn_combine_kernel<TO, D>;
  const int64_t threads = (int64_t)p.bh * p.n_q * (D / 4);
  return hipLaunchKernel(reinterpret_cast<const void*>(comb), dim3((unsigned)((threads + 255) / 256)),
                         dim3(256), args, 0, stream);
}

template <typename T, typename TO, int D>
static hipError_t launch_fwd_dt(const FwdParams& p, bool causal, hipStream_t stream) {
  constexpr int QT = FwdShape<T, D>::QT, BK = FwdShape<T, D>::BK;
  return causal ? launch_fwd_impl<T, TO, D, QT, BK, true>(p, stream)
                : launch_fwd_impl<T, TO, D, QT, BK, false>(p, stream);
}

template <typename T, int D>
static hipError_t launch_fwd_out(const FwdParams& p, bool causal, bool out_f32, hipStream_t stream) {
  return out_f32 ? launch_fwd_dt<T, float, D>(p, causal, stream) : launch_fwd_dt<T, T, D>(p, causal, stream);
}

hipError_t launch_fwd(const FwdParams& p, int dtype, int d, bool causal, bool out_f32,
                      hipStream_t stream) {
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
