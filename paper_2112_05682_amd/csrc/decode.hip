// Decode-shaped forward: a small group of queries (n_q <= 64 per batch and
// head) against a long key sequence.  This is the paper's single-query
// algorithm (Section 2, stabilised by the running maximum of Section 3)
// generalised to a query group, with the keys split into ranges whose
// summaries are combined afterwards (Section 4): each workgroup is one wave
// that streams one key range of one (batch, head) through LDS and keeps the
// running numerator, denominator and maximum of every query of the group.
//
// The work is bound by HBM (K and V are read once: 4 d bytes per key for
// 16-bit inputs against 4 d n_q flops), so the kernel is shaped for bytes in
// flight rather than for matrix throughput: one wave per workgroup, a
// two-stage LDS ring of asynchronous copies per wave, and enough workgroups
// per CU (the ring is 36 KiB, 32 KiB with swizzled rows) to keep about
// 64 KiB of copies in flight per CU.  The scores and the weighted values still go through MFMA with the
// query group padded to 32 or 64 columns: at n_q <= 64 the padded matrix work
// stays below the HBM time.
#include <type_traits>

#include "device.hpp"
#include "kernels.hpp"

namespace mea {

namespace dec {
// Tile geometry for head dimension D: BK keys per tile, LDS rows of D
// features plus one 16-byte pad slot (row and transposing reads then touch
// distinct banks), the copies of a tile as NCOPY 1 KiB wave copies (the slots
// past the tile's rows are a dead tail inside the tile's LDS space).
template <int D>
struct Cfg {
  static constexpr int BK = D == 64 ? 64 : 32;
  static constexpr int SPR = D / 8 + 1;  // 16-byte slots per LDS row
  static constexpr int RSB = 16 * SPR;   // bytes per LDS row
  static constexpr int NSLOT = BK * SPR;
  static constexpr int NCOPY = (NSLOT + 63) / 64;
  static constexpr int TILEB = NCOPY * 1024;
  static constexpr int NSTAGE = 2;
  static constexpr int STAGEB = 2 * TILEB;  // K tile, V tile
  static_assert(BK * RSB <= TILEB, "rows fit the tile");
};
// The same tiles in unpadded 256-byte rows (d = 128) whose 16-byte chunks are
// XOR-swizzled: the physical chunk of logical chunk x in row r is
// x ^ swz(r), with r & 15 for K (row reads) and (r & 3) << 2 for V
// (transposing reads), so that both touch distinct banks.  A copy moves RPU = 4
// rows; the K swizzle repeats every KP = 4 copies and the V swizzle within
// one, so a lane needs KP + 1 copy offsets instead of the padded layout's
// 4 NCOPY (row, column and both offsets per copy).
struct Swz128 {
  static constexpr int BK = 32, ROWB = 256, CPR = 16, RPU = 4, KP = 4;
  static constexpr int NCOPY = BK * ROWB / 1024;
  static constexpr int TILEB = BK * ROWB;
  static constexpr int NSTAGE = 2;
  static constexpr int STAGEB = 2 * TILEB;
  __device__ static __forceinline__ int swz_k(int r) { return r & 15; }
  __device__ static __forceinline__ int swz_v(int r) { return (r & 3) << 2; }
  static_assert(NCOPY % KP == 0 && RPU * KP == 16, "copy geometry");
};
}  // namespace dec

// Top-left causal (key j visible to query i iff j <= i): only the first n_q
// keys can be visible to a group of n_q queries.
__host__ __device__ inline int64_t decode_keys(int64_t n_q, int64_t n_k, bool causal) {
  return causal && n_k > n_q ? n_q : n_k;
}

// One wave: queries 0 .. 32 QT - 1 of (batch, head) bh against keys
// [split * keys_per_split, ...).  Scores in the orientation S^T = K Q^T (lane =
// query, registers = keys, K rows read in the perm32 order so that the
// weights convert in place into the B operand of O^T += V^T P^T).
// With two query sub-tiles at d = 128 the padded layout's copy offsets (36
// registers) spilled and were reloaded in the tile loop; that variant uses the
// swizzled rows (SWZ).  The others keep the padded rows, whose reads need no
// per-fragment address arithmetic.
template <typename T, typename TO, int D, int QT, bool CAUSAL>
__global__ __launch_bounds__(64) void attn_decode_kernel(FwdParams p) {
  constexpr bool SWZ = D == 128 && QT == 2;
  using C = std::conditional_t<SWZ, dec::Swz128, dec::Cfg<D>>;
  using P = dec::Cfg<D>;
  using S = dec::Swz128;
  constexpr int BK = C::BK, NKT = BK / 32, KC = D / 16, NDT = D / 32, NPC = BK / 16;
  constexpr int RS = P::RSB / 2;  // padded LDS row stride in elements
  __shared__ __align__(16) unsigned char smem[C::NSTAGE * C::STAGEB];

  const int lane = threadIdx.x;
  const int h = lane >> 5, c = lane & 31;
  const int split = blockIdx.x % p.n_splits;
  const int bh = blockIdx.x / p.n_splits;

  const T* __restrict__ qg = static_cast<const T*>(p.q) + head_base(p.sq, bh, p.heads);
  const T* __restrict__ kg = static_cast<const T*>(p.k) + head_base(p.sk, bh, p.heads);
  const T* __restrict__ vg = static_cast<const T*>(p.v) + head_base(p.sv, bh, p.heads);

  // Keys visible to this (batch, head): n_k, or the batch's valid length
  // (key padding); with the causal mask at most the first n_q of them.
  const int64_t n_keys = decode_keys(p.n_q, valid_keys(p.kv_len, bh, p.heads, p.n_k), CAUSAL);
  const int64_t kb = (int64_t)split * p.keys_per_split;
  int64_t ke = kb + p.keys_per_split;
  if (ke > n_keys) ke = n_keys;
  const int n_tiles = kb < ke ? (int)((ke - kb + BK - 1) / BK) : 0;

  // Q^T as B operands: lane (h, c) holds query 32 t + c, features 16 kc + 8 h ..
  Frag<T> qf[QT][KC];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const int64_t query = 32 * t + c;
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
      if (query < p.n_q) {
        qf[t][kc] = *reinterpret_cast<const Frag<T>*>(qg + query * p.sq.r + 16 * kc + 8 * h);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[t][kc][e] = (T)0.0f;
      }
    }
  }

  // Padded rows: copy u of a tile moves lane slots 64 u + lane: row
  // slot / SPR, 16-byte chunk slot % SPR (the pad slot gets a copy of the last
  // chunk); slots past the tile's rows repeat its last slot.  The row and the
  // byte column of each copy are computed once, and the byte offsets within a
  // tile of K and of V (row strides < 2^24 elements, checked on the host).
  // Swizzled rows: copy u moves rows 4 u .. 4 u + 3, lane l writing physical
  // chunk l % 16 of row 4 u + l / 16; the K offset of copy u is that of copy
  // u % KP (plus a scalar shift of 16 (u / KP) rows), the V offset is the same
  // for every copy.
  constexpr int NPAD = SWZ ? 1 : C::NCOPY;
  int urow[NPAD];
  unsigned ucol[NPAD], ukoff[NPAD], uvoff[NPAD];
  unsigned skoff[S::KP], svoff = 0;
  const int lrow = lane / S::CPR, lx = lane % S::CPR;
  if constexpr (SWZ) {
#pragma unroll
    for (int b = 0; b < S::KP; ++b) {
      const int row = S::RPU * b + lrow;
      skoff[b] = 2u * ((unsigned)row * (unsigned)p.sk.r + 8u * (unsigned)(lx ^ S::swz_k(row)));
    }
    svoff = 2u * ((unsigned)lrow * (unsigned)p.sv.r + 8u * (unsigned)(lx ^ S::swz_v(lrow)));
  } else {
#pragma unroll
    for (int u = 0; u < NPAD; ++u) {
      int slot = 64 * u + lane;
      if (slot >= P::NSLOT) slot = P::NSLOT - 1;
      const int ch = slot % P::SPR;
      urow[u] = slot / P::SPR;
      ucol[u] = (unsigned)(16 * (ch < P::SPR - 1 ? ch : P::SPR - 2));
      ukoff[u] = (unsigned)urow[u] * (unsigned)(2 * p.sk.r) + ucol[u];
      uvoff[u] = (unsigned)urow[u] * (unsigned)(2 * p.sv.r) + ucol[u];
    }
  }
  auto copy_tile = [&](int j) __attribute__((always_inline)) {
    const int64_t k0 = kb + (int64_t)j * BK;
    unsigned char* st = smem + (j % C::NSTAGE) * C::STAGEB;
    const unsigned kl = lds_addr(st), vl = lds_addr(st + C::TILEB);
    const bool full = k0 + BK <= ke;
    if constexpr (SWZ) {
      if (full) {
#pragma unroll
        for (int u = 0; u < C::NCOPY; ++u) {
          copy_to_lds16_sb<true>(kg + (k0 + 16 * (u / S::KP)) * p.sk.r, skoff[u % S::KP],
                                 __builtin_amdgcn_readfirstlane(kl + 1024 * u));
          copy_to_lds16_sb<true>(vg + (k0 + S::RPU * u) * p.sv.r, svoff, __builtin_amdgcn_readfirstlane(vl + 1024 * u));
        }
      } else {
        // Ragged last tile: rows past the range repeat its last key (finite
        // values, masked below).
#pragma unroll
        for (int u = 0; u < C::NCOPY; ++u) {
          const int row = S::RPU * u + lrow;
          int64_t key = k0 + row;
          if (key > ke - 1) key = ke - 1;
          copy_to_lds16<true>(kg + key * p.sk.r + 8 * (lx ^ S::swz_k(row)), __builtin_amdgcn_readfirstlane(kl + 1024 * u));
          copy_to_lds16<true>(vg + key * p.sv.r + 8 * (lx ^ S::swz_v(row)), __builtin_amdgcn_readfirstlane(vl + 1024 * u));
        }
      }
    } else if (full) {
#pragma unroll
      for (int u = 0; u < C::NCOPY; ++u) {
        copy_to_lds16_sb<true>(kg + k0 * p.sk.r, ukoff[u], __builtin_amdgcn_readfirstlane(kl + 1024 * u));
        copy_to_lds16_sb<true>(vg + k0 * p.sv.r, uvoff[u], __builtin_amdgcn_readfirstlane(vl + 1024 * u));
      }
    } else {
#pragma unroll
      for (int u = 0; u < C::NCOPY; ++u) {
        int64_t key = k0 + urow[u];
        if (key > ke - 1) key = ke - 1;
        copy_to_lds16<true>(reinterpret_cast<const unsigned char*>(kg + key * p.sk.r) + ucol[u],
                            __builtin_amdgcn_readfirstlane(kl + 1024 * u));
        copy_to_lds16<true>(reinterpret_cast<const unsigned char*>(vg + key * p.sv.r) + ucol[u],
                            __builtin_amdgcn_readfirstlane(vl + 1024 * u));
      }
    }
  };

  const float cl2 = p.scale_log2;
  const int krow = perm32(c);
  float m_run[QT], l_run[QT];
  f32x16 acc[QT][NDT];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    m_run[t] = -INFINITY;
    l_run[t] = 0.0f;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[t][dt][r] = 0.0f;
  }

  if (n_tiles > 0) copy_tile(0);
  if (n_tiles > 1) copy_tile(1);
  for (int j = 0; j < n_tiles; ++j) {
    // Tile j has landed once at most the copies of tile j + 1 are in flight.
    if (j + 1 < n_tiles) wait_global_loads_upto<2 * C::NCOPY>();
    else wait_global_loads();
    const unsigned char* st = smem + (j % C::NSTAGE) * C::STAGEB;
    const T* ks = reinterpret_cast<const T*>(st);
    const T* vs = reinterpret_cast<const T*>(st + C::TILEB);
    const int64_t k0 = kb + (int64_t)j * BK;

    // S^T = K Q^T for the tile (one K fragment serves every query sub-tile).
    f32x16 s[QT][NKT];
#pragma unroll
    for (int t = 0; t < QT; ++t)
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[t][kt][r] = 0.0f;
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int kc = 0; kc < KC; ++kc) {
        const int row = 32 * kt + krow;
        Frag<T> kf;
        if constexpr (SWZ)
          kf = *reinterpret_cast<const Frag<T>*>(reinterpret_cast<const unsigned char*>(ks) + row * S::ROWB +
                                                   16 * ((2 * kc + h) ^ S::swz_k(row)));
        else
          kf = lds_frag<T>(ks + row * RS + 16 * kc + 8 * h);
#pragma unroll
        for (int t = 0; t < QT; ++t) s[t][kt] = mma(kf, qf[t][kc], s[t][kt]);
      }

    // Mask keys past the range (ragged tile) and, causal, keys after the query.
    if (CAUSAL || k0 + BK > ke) {
#pragma unroll
      for (int t = 0; t < QT; ++t) {
        int64_t lim = ke - k0;  // keys k0 + x with x < lim are in range
        if (CAUSAL && 32 * t + c + 1 - k0 < lim) lim = 32 * t + c + 1 - k0;
#pragma unroll
        for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (32 * kt + permuted_row(r, h) >= lim) s[t][kt][r] = -INFINITY;
      }
    }

    // Online softmax per query (lane), with the lazy reference m_run (in units
    // of c S): it rises only when a score exceeds it by more than
    // kRescaleSlack powers of two, so most tiles skip the rescale of the
    // running numerator and denominator (both share the reference, so the
    // result is the same).  A query with no visible key yet keeps
    // m_run = -inf and offset 0 (its weights are 2^-inf = 0).
    Frag<T> pf[QT][NPC];
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[t][kt][r]);
      const float mx_c = xhalf_max(mx) * cl2;
      const bool raise = mx_c > m_run[t] + kRescaleSlack;
      if (__builtin_amdgcn_ballot_w64(raise)) {
        const float m_new = raise ? mx_c : m_run[t];
        // 0 on a first raise; 1 for a lane that does not raise (also one
        // still at -inf, where the difference would be NaN).
        const float alpha = raise ? fast_exp2(m_run[t] - m_new) : 1.0f;
        m_run[t] = m_new;
        l_run[t] *= alpha;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[t][dt][r] *= alpha;
      }
      const float neg = m_run[t] == -INFINITY ? 0.0f : -m_run[t];
#pragma unroll
      for (int pc = 0; pc < NPC; ++pc) {
        float w8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) w8[e] = fast_exp2(fmaf(s[t][pc >> 1][8 * (pc & 1) + e], cl2, neg));
        pf[t][pc] = to_frag<T>(w8);
        l_run[t] = tree_sum<8>(w8, l_run[t]);
      }
    }

    // O^T += V^T P^T (one V fragment serves every query sub-tile); swizzled
    // rows: the transposing reads of lds_col_frag with the V swizzle applied.
    const int g4 = lane >> 4, i4 = lane & 15;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int pc = 0; pc < NPC; ++pc) {
        Frag<T> vf;
        if constexpr (SWZ) {
          const unsigned char* vb = reinterpret_cast<const unsigned char*>(vs);
          const int row = 16 * pc + 8 * (g4 >> 1) + (i4 >> 2);
          const int colb = 2 * (32 * dt + 16 * (g4 & 1) + 4 * (i4 & 3));
          const v4s_t lo = lds_read_tr16(vb + row * S::ROWB + (((colb >> 4) ^ S::swz_v(row)) << 4) + (colb & 15));
          const v4s_t hi =
              lds_read_tr16(vb + (row + 4) * S::ROWB + (((colb >> 4) ^ S::swz_v(row + 4)) << 4) + (colb & 15));
          typedef short v8s_t __attribute__((ext_vector_type(8)));
          v8s_t r8;
          r8[0] = lo[0]; r8[1] = lo[1]; r8[2] = lo[2]; r8[3] = lo[3];
          r8[4] = hi[0]; r8[5] = hi[1]; r8[6] = hi[2]; r8[7] = hi[3];
          vf = __builtin_bit_cast(Frag<T>, r8);
        } else {
          vf = lds_col_frag<T>(vs, RS, 16 * pc, 32 * dt, lane);
        }
#pragma unroll
        for (int t = 0; t < QT; ++t) acc[t][dt] = mma(vf, pf[t][pc], acc[t][dt]);
      }

    // The stage is free once its reads have returned; refill it with tile j + 2.
    if (j + 2 < n_tiles) {
      wait_lds_reads();
      copy_tile(j + 2);
    }
  }

  // Epilogue: the two lane halves hold disjoint keys of the same query.
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const float l_tot = xhalf_sum(l_run[t]);
    const int64_t row = 32 * t + c;
    if (row >= p.n_q) continue;
    if (p.n_splits == 1) {
      const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;  // no visible key: o = 0
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
        p.lse[(size_t)bh * p.n_q + row] = l_tot > 0.0f ? (m_run[t] + __log2f(l_tot)) * 0.6931471805599453f : -INFINITY;
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
        p.part_m[prow] = m_run[t];  // reference, log2 units (scaled); -inf if the range has no visible key
        p.part_l[prow] = l_tot;
      }
    }
  }
}

template <typename T, typename TO, int D>
static hipError_t launch_decode_dt(const FwdParams& p, bool causal, hipStream_t stream) {
  FwdParams pc = p;
  void* args[] = {&pc};
  const dim3 grid((unsigned)((int64_t)p.bh * p.n_splits)), block(64);
  if (p.n_q <= 32) {
    auto k = causal ? attn_decode_kernel<T, TO, D, 1, true> : attn_decode_kernel<T, TO, D, 1, false>;
    return hipLaunchKernel(reinterpret_cast<const void*>(k), grid, block, args, 0, stream);
  }
  auto k = causal ? attn_decode_kernel<T, TO, D, 2, true> : attn_decode_kernel<T, TO, D, 2, false>;
  return hipLaunchKernel(reinterpret_cast<const void*>(k), grid, block, args, 0, stream);
}

template <typename T, int D>
static hipError_t launch_decode_out(const FwdParams& p, bool causal, bool out_f32, hipStream_t stream) {
  return out_f32 ? launch_decode_dt<T, float, D>(p, causal, stream) : launch_decode_dt<T, T, D>(p, causal, stream);
}

hipError_t launch_decode(const FwdParams& p, int dtype, int d, bool causal, bool out_f32, hipStream_t stream) {
  switch (dtype * 1000 + d) {
    case 1 * 1000 + 64: return launch_decode_out<_Float16, 64>(p, causal, out_f32, stream);
    case 1 * 1000 + 128: return launch_decode_out<_Float16, 128>(p, causal, out_f32, stream);
    case 2 * 1000 + 64: return launch_decode_out<__bf16, 64>(p, causal, out_f32, stream);
    case 2 * 1000 + 128: return launch_decode_out<__bf16, 128>(p, causal, out_f32, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace mea
