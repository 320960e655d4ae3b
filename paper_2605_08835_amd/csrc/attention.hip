// Multi-head attention O = softmax(Q K^T * scale) V for self-attention over
// image tokens and cross-attention to the text context.
//
// bf16: flash-style (online softmax, Dao et al. 2022) on MFMA.  Each wave owns
// 32 queries; a block of 4 waves shares LDS-staged tiles of 64 keys.  The
// scores are computed transposed, S^T = K Q^T, so that a lane holds one
// query's scores in registers: the softmax row statistics need a single
// cross-lane exchange and the rescale of the (also transposed) output
// accumulator O^T = V^T P^T is a per-lane multiply.  The probabilities feed
// the second MFMA straight from registers; the keys of each 16-key MFMA
// slice are permuted to match the accumulator layout, and V^T is read from
// LDS with the same permutation.
//
// Softmax bookkeeping is kept off the vector ALU where the MFMAs can carry
// it, since at SD head widths (d = 40) the exp and its companions, not the
// products, bound the kernel:
//  * Q arrives pre-scaled by scale * log2(e) (the projection GEMM's epilogue
//    multiplies before its one rounding), so a score is already a base-2
//    exponent and each probability is one exp2.  Unscaled Q is also
//    accepted; then each score takes one fma more.
//  * With pre-scaled Q, the running maximum m is subtracted inside the QK^T
//    product when the head width leaves a spare padding column
//    (d % 16 != 0): K carries a 1 in column d and Q carries -m there (m kept
//    bf16-representable, so the product is exact).
//  * The row sum of P comes out of the PV product when V^T has a spare
//    padding row (d % 32 != 0): that row of V^T is 1 for every valid key.
//  * m only moves when a tile's maximum exceeds it by more than 8 (so no
//    probability exceeds 2^8); the rescale of the accumulators, the rare
//    case after the first tile, is a wave-uniform branch.  The result is
//    the same softmax: any m with no overflow gives the same quotient.
// fp32: one thread per query, K/V tiles in LDS, fp32 online softmax.
#include "device_common.h"
#include "kernels.h"

namespace sd {

namespace fa {
constexpr int KT = 64;        // keys per tile
constexpr float TAU = 8.0f;   // lazy-rescale threshold (log2 units)
}

__device__ inline float bf16_rne(float x) { return (float)(bf16)x; }

// v op v of lane l ^ 32: one lane-half swap instead of a trip through LDS.
// (The builtin exists only for the device pass; the host pass never runs it.)
__device__ inline float2 xor32_pair(float v) {
#if defined(__HIP_DEVICE_COMPILE__)
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return make_float2(__uint_as_float(r[0]), __uint_as_float(r[1]));
#else
  return make_float2(v, v);
#endif
}
__device__ inline float xor32_max(float v) {
  const float2 p = xor32_pair(v);
  return fmaxf(p.x, p.y);
}
__device__ inline float xor32_sum(float v) {
  const float2 p = xor32_pair(v);
  return p.x + p.y;
}

template <bool B>
struct BC {
  static constexpr bool value = B;
};

template <int V>
struct IC {
  static constexpr int value = V;
};
template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(IC<I>{});
    static_for<I + 1, N>(f);
  }
}

__device__ inline bf16x8 ld16(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }

// Online-softmax step on one 64-key tile of S^T (NKT = 2), or on its first
// 32 keys (NKT = 1: a last tile of at most 32 keys).  On entry s holds the raw
// products: base-2 logits minus m when MF, base-2 logits when QS, plain
// q.k otherwise.  Moves m where the tile exceeds it by more than TAU,
// rescales the accumulators then, and leaves P = exp2(logit - m) in s.  SF:
// the row sum comes out of the PV product, else it is added up here.
template <int NJ, int ND, bool QS, bool MF, bool SF, bool TAIL, int NKT = 2>
__device__ __forceinline__ void softmax_tile(f32x16 (&s)[2], f32x16 (&o)[ND], bf16x8 (&qf)[NJ], float& m_run,
                                             float& l_run, bool first, int kvalid, int lh, int d, float sl2) {
  using namespace fa;
  if constexpr (!QS) {
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kt][r] = fmaf(s[kt][r], sl2, -m_run);
  } else if constexpr (!MF) {  // no spare column: subtract m here
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kt][r] -= m_run;
  }
  if constexpr (TAIL) {  // keys at or past kvalid; compared as immediates against one register
    const int lim = kvalid - 4 * lh;
    static_for<0, 16 * NKT>([&](auto I) {
      constexpr int kt = I.value / 16, r = I.value % 16;
      if (kt * 32 + 8 * (r >> 2) + (r & 3) >= lim) s[kt][r] = -1e30f;
    });
  }
  float mt = -1e30f;
#pragma unroll
  for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
    for (int r = 0; r < 16; ++r) mt = fmaxf(mt, s[kt][r]);
  mt = xor32_max(mt);
  const bool need = first || mt > TAU;
  if (__any(need)) {
    // move m to the (bf16-rounded) tile maximum where needed
    float delta = 0.f;
    if (need) {
      const float mn = bf16_rne(m_run + mt);
      delta = mn - m_run;
      m_run = mn;
    }
    // (nothing has accumulated before the first tile; its delta may be any
    // size, so alpha is not evaluated there)
    const float alpha = first ? 0.f : __builtin_amdgcn_exp2f(-delta);
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kt][r] -= delta;
    l_run *= alpha;
#pragma unroll
    for (int t = 0; t < ND; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[t][r] *= alpha;
    if constexpr (MF) {
      const bf16 nm = (bf16)(-m_run);
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (16 * j + 8 * lh + e == d) qf[j][e] = nm;
    }
  }
#pragma unroll
  for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
    for (int r = 0; r < 16; ++r) s[kt][r] = __builtin_amdgcn_exp2f(s[kt][r]);
  if constexpr (!SF) {
    float ps = 0.f;
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) ps += s[kt][r];
    l_run += ps;
  }
}

// D16: head width rounded up to 16 (the QK^T reduction); DP: rounded up to
// 32 (the PV output rows).  QS: Q holds base-2 logit units (q * scale *
// log2 e, written so by the projection GEMM).  MF (needs QS): d < D16, the
// max rides in column d of the QK^T product.  SF: d < DP, the row sum rides
// in row d of the PV product.  V is stored transposed per image
// ([channel][token], as the projection GEMM writes it), so a V^T tile is
// staged with 16-byte loads and stores.
template <int D16, bool QS, bool MF, bool SF, int NW, int QG>
__global__ __launch_bounds__(64 * NW, D16 <= 128 ? 2 : 1) void attn_bf16_kernel(AttnArgs a) {
  using namespace fa;
  static_assert(QS || !MF, "the max can ride in the product only with pre-scaled queries");
  constexpr int NJ = D16 / 16, DP = (D16 + 31) / 32 * 32, ND = DP / 32;
  constexpr int LDK = D16 + 8, LDV = KT + 8, NT = 64 * NW;
  constexpr int KCH = KT * (D16 / 8), VCH = DP * (KT / 8);  // 16-byte chunks per tile
  constexpr int KPT = (KCH + NT - 1) / NT, VPT = (VCH + NT - 1) / NT;  // ... per thread
  // Double-buffered K and V^T tiles; the next tile is fetched into registers
  // while the current one feeds the MFMAs.
  __shared__ __attribute__((aligned(16))) bf16 Ks[2][KT * LDK];
  __shared__ __attribute__((aligned(16))) bf16 Vt[2][DP * LDV];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int img = blockIdx.z, head = blockIdx.y;
  const int qb = blockIdx.x * (32 * NW * QG) + wave * (32 * QG);
  const int kvimg = a.kv_index ? a.kv_index[img] : img;
  const int hd = head * a.d;
  const bf16* Q = reinterpret_cast<const bf16*>(a.q) + (long)img * a.q_img + hd;
  const bf16* K = reinterpret_cast<const bf16*>(a.k) + (long)kvimg * a.k_img + hd;
  const bf16* V = reinterpret_cast<const bf16*>(a.v) + (long)kvimg * a.v_img + (long)hd * a.v_ld;
  const int lq = lane & 31, lh = lane >> 5;
  const int d = a.d;
  const float sl2 = a.scale * 1.4426950408889634f;  // used when !QS

  // Q^T fragment (B operand): query qb + lq, head dims 16 j + 8 lh + [0, 8);
  // column d (when MF) holds -m.
  // QG groups of 32 queries per wave share every K and V fragment read.
  bf16x8 qf[QG][NJ];
#pragma unroll
  for (int g = 0; g < QG; ++g) {
    const int q = qb + 32 * g + lq;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int dd = 16 * j + 8 * lh;
      const bf16x8 z = {};
      qf[g][j] = (q < a.Nq && dd < d) ? ld16(Q + (long)q * a.q_ld + dd) : z;
    }
  }
  f32x16 o[QG][ND];
#pragma unroll
  for (int g = 0; g < QG; ++g)
#pragma unroll
    for (int t = 0; t < ND; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[g][t][r] = 0.f;
  float m_run[QG], l_run[QG];
#pragma unroll
  for (int g = 0; g < QG; ++g) m_run[g] = l_run[g] = 0.f;
  const bool vvec = (a.v_ld & 7) == 0;

  // PF2 (the narrow heads with the max in the product, d = 40 for SD):
  // two register sets, the tile after next fetched while this one is
  // computed and the next one (fetched a tile earlier) staged into LDS, so a
  // fetch has two tiles of time to land (measured +4 % at d = 40; at the
  // wider heads it measured slower or ran out of registers).  Otherwise the
  // next tile is fetched during this one, into the single set it needs.
  constexpr bool PF2 = QG == 2 && D16 == 48 && MF;
  bf16x8 rk0[KPT], rv0[VPT], rk1[KPT], rv1[VPT];
  auto fetch = [&](int k0, bf16x8 (&rk)[KPT], bf16x8 (&rv)[VPT]) {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int idx = tid + NT * i;
      const int key = idx / (D16 / 8), dc = (idx - key * (D16 / 8)) * 8;
      bf16x8 v = {};
      if (idx < KCH && k0 + key < a.Nk) {
        if (dc < d)
          v = ld16(K + (long)(k0 + key) * a.k_ld + dc);
        else if (MF && dc == d)  // the column that subtracts m
          v[0] = (bf16)1.0f;
      }
      rk[i] = v;
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int idx = tid + NT * i;
      const int dd = idx / (KT / 8), kc = (idx - dd * (KT / 8)) * 8;
      const int k = k0 + kc;
      bf16x8 v = {};
      if (idx < VCH && dd < d && k < a.Nk) {
        const bf16* src = V + (long)dd * a.v_ld + k;
        if (vvec && k + 8 <= a.Nk) {
          v = ld16(src);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (k + e < a.Nk) v[e] = src[e];
        }
      } else if (SF && idx < VCH && dd == d) {  // ones row: PV also sums P
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (k + e < a.Nk) v[e] = (bf16)1.0f;
      }
      rv[i] = v;
    }
  };
  auto stage = [&](int b, const bf16x8 (&rk)[KPT], const bf16x8 (&rv)[VPT]) {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int idx = tid + NT * i;
      const int key = idx / (D16 / 8), dc = (idx - key * (D16 / 8)) * 8;
      if (idx < KCH) *reinterpret_cast<bf16x8*>(&Ks[b][key * LDK + dc]) = rk[i];
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int idx = tid + NT * i;
      const int dd = idx / (KT / 8), kc = (idx - dd * (KT / 8)) * 8;
      if (idx < VCH) *reinterpret_cast<bf16x8*>(&Vt[b][dd * LDV + kc]) = rv[i];
    }
  };

  // Heads with the max in the product (d = D16 - 8, a compile-time width):
  // the padding of K (the ones column d) and of V^T (the ones row d, then
  // zero rows) is the same for every tile, so it is written into both LDS
  // buffers once, and a tile moves only its d / 8 data chunks per key and
  // its d rows of V^T (the general fetch spent more vector instructions on
  // addressing and masks than the softmax on its maxima).  Keys past the
  // end load as zeros; the ones row keeps 1 there, which the masked
  // probabilities (exactly 0) multiply away, so the sums are unchanged.
  // The same holds for every pre-scaled variant, whose width is fixed at
  // compile time too (d = D16 when the max does not ride in the product):
  // no K padding then, and the V^T ones row only when the sum rides in PV.
  // (Not at 128 and above 160, where the extra registers spill.)
  constexpr bool FAST = QS && (D16 <= 96 || D16 == 160);
  constexpr int DV = MF ? D16 - 8 : D16, CK = DV / 8;
  constexpr int KV = KT * CK, VV = DV * (KT / 8);  // data chunks per tile
  constexpr int KPF = (KV + NT - 1) / NT, VPF = (VV + NT - 1) / NT;
  static_assert(!FAST || (KPF <= KPT && VPF <= VPT), "the data chunks fit the fetch registers");
  auto fetch_data = [&](int k0, bf16x8 (&rk)[KPT], bf16x8 (&rv)[VPT]) {
#pragma unroll
    for (int i = 0; i < KPF; ++i) {
      const int idx = tid + NT * i;
      if (KV % NT == 0 || idx < KV) {
        const int key = idx / CK, c = idx - key * CK;
        bf16x8 v = {};
        if (k0 + key < a.Nk) v = ld16(K + (long)(k0 + key) * a.k_ld + 8 * c);
        rk[i] = v;
      }
    }
#pragma unroll
    for (int i = 0; i < VPF; ++i) {
      const int idx = tid + NT * i;
      if (VV % NT == 0 || idx < VV) {
        const int dd = idx / (KT / 8), kc = (idx - dd * (KT / 8)) * 8;
        const int k = k0 + kc;
        const bf16* src = V + (long)dd * a.v_ld + k;
        bf16x8 v = {};
        if (vvec && k + 8 <= a.Nk) {
          v = ld16(src);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (k + e < a.Nk) v[e] = src[e];
        }
        rv[i] = v;
      }
    }
  };
  auto stage_data = [&](int b, const bf16x8 (&rk)[KPT], const bf16x8 (&rv)[VPT]) {
#pragma unroll
    for (int i = 0; i < KPF; ++i) {
      const int idx = tid + NT * i;
      if (KV % NT == 0 || idx < KV) {
        const int key = idx / CK, c = idx - key * CK;
        *reinterpret_cast<bf16x8*>(&Ks[b][key * LDK + 8 * c]) = rk[i];
      }
    }
#pragma unroll
    for (int i = 0; i < VPF; ++i) {
      const int idx = tid + NT * i;
      if (VV % NT == 0 || idx < VV) {
        const int dd = idx / (KT / 8), kc = (idx - dd * (KT / 8)) * 8;
        *reinterpret_cast<bf16x8*>(&Vt[b][dd * LDV + kc]) = rv[i];
      }
    }
  };
  if constexpr (FAST) {
    // K: chunk DV of every key of both buffers (the ones column; none when
    // DV = D16); V^T: rows DV..DP-1 of both
    if constexpr (MF)
      for (int c = tid; c < 2 * KT; c += NT) {
        bf16x8 v = {};
        v[0] = (bf16)1.0f;
        *reinterpret_cast<bf16x8*>(&Ks[c / KT][(c % KT) * LDK + DV]) = v;
      }
    constexpr int PR = (DP - DV) * (KT / 8);  // padding chunks per buffer
    for (int c = tid; c < 2 * PR; c += NT) {
      const int b = c / PR, r = c - b * PR, dd = DV + r / (KT / 8), kc = (r % (KT / 8)) * 8;
      bf16x8 v = {};
      if (SF && dd == DV)
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = (bf16)1.0f;
      *reinterpret_cast<bf16x8*>(&Vt[b][dd * LDV + kc]) = v;
    }
  }
  // A tile known to be full, with 16-byte aligned V^T rows: no bounds checks
  // and no element-wise fallback, so the loop that uses it holds only the
  // 16-byte loads (a fallback's scalar loads into temporaries make the
  // compiler wait for every outstanding load before the products).
  auto fetch_full = [&](int k0, bf16x8 (&rk)[KPT], bf16x8 (&rv)[VPT]) {
#pragma unroll
    for (int i = 0; i < KPF; ++i) {
      const int idx = tid + NT * i;
      if (KV % NT == 0 || idx < KV) {
        const int key = idx / CK, c = idx - key * CK;
        rk[i] = ld16(K + (long)(k0 + key) * a.k_ld + 8 * c);
      }
    }
#pragma unroll
    for (int i = 0; i < VPF; ++i) {
      const int idx = tid + NT * i;
      if (VV % NT == 0 || idx < VV) {
        const int dd = idx / (KT / 8), kc = (idx - dd * (KT / 8)) * 8;
        rv[i] = ld16(V + (long)dd * a.v_ld + k0 + kc);
      }
    }
  };
  auto fetch_any = [&](int k0, bf16x8 (&rk)[KPT], bf16x8 (&rv)[VPT]) {
    if constexpr (FAST)
      fetch_data(k0, rk, rv);
    else
      fetch(k0, rk, rv);
  };
  auto stage_any = [&](int b, int, const bf16x8 (&rk)[KPT], const bf16x8 (&rv)[VPT]) {
    if constexpr (FAST)
      stage_data(b, rk, rv);
    else
      stage(b, rk, rv);
  };

  fetch_any(0, rk0, rv0);
  stage_any(0, 0, rk0, rv0);
  if (PF2 && KT < a.Nk) fetch_any(KT, rk1, rv1);
  __syncthreads();
  // One 64-key tile; the last tile, if partial, is a separate instance so
  // the full tiles carry no masking code.
  // fk / fv: the set to fetch the tile after next into; sk / sv: the set
  // holding the next tile, staged at the end.
  // FULL: the tile it fetches is full and V^T is aligned (FAST heads only).
  // HALF (a tail of at most 32 keys): only the first 32-key block of S^T and
  // the first two PV slices; the keys past it were masked to P = 0, so the
  // products skipped added exact zeros and the result is the same.
  auto tile = [&](auto tl, auto ff, int k0, int it, bf16x8 (&fk)[KPT], bf16x8 (&fv)[VPT], bf16x8 (&sk)[KPT],
                  bf16x8 (&sv)[VPT], auto hf) {
    constexpr bool TAIL = decltype(tl)::value, FULL = decltype(ff)::value, HALF = decltype(hf)::value;
    static_assert(TAIL || !HALF, "only a tail tile is halved");
    constexpr int NKT = HALF ? 1 : 2;
    const int b = it & 1;
    const bool more = k0 + KT < a.Nk;
    if constexpr (FULL) {
      fetch_full(k0 + (PF2 ? 2 : 1) * KT, PF2 ? fk : sk, PF2 ? fv : sv);
    } else if constexpr (PF2) {
      if (k0 + 2 * KT < a.Nk) fetch_any(k0 + 2 * KT, fk, fv);
    } else {
      if (more) fetch_any(k0 + KT, sk, sv);
    }
    const bf16* Kb = Ks[b];
    const bf16* Vb = Vt[b];

    // S^T tiles: rows = keys kt*32 + 8(r/4) + 4 lh + r%4, col = query.
    f32x16 s[QG][2];
#pragma unroll
    for (int g = 0; g < QG; ++g)
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[g][kt][r] = 0.f;
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const bf16x8 kf = ld16(&Kb[(kt * 32 + lq) * LDK + 16 * j + 8 * lh]);
#pragma unroll
        for (int g = 0; g < QG; ++g) s[g][kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[g][j], s[g][kt], 0, 0, 0);
      }
#pragma unroll
    for (int g = 0; g < QG; ++g)
      softmax_tile<NJ, ND, QS, MF, SF, TAIL, NKT>(s[g], o[g], qf[g], m_run[g], l_run[g], it == 0, a.Nk - k0, lh, d,
                                                  sl2);

    // O^T += V^T P^T over four 16-key slices.  Slot (lh, i) of slice u is
    // key 16u + 8(i/4) + 4 lh + i%4, i.e. register 8(u%2) + i of S^T tile u/2.
#pragma unroll
    for (int u = 0; u < 2 * NKT; ++u) {
      bf16x8 pf[QG];
#pragma unroll
      for (int g = 0; g < QG; ++g)
#pragma unroll
        for (int i = 0; i < 8; ++i) pf[g][i] = (bf16)s[g][u >> 1][8 * (u & 1) + i];
#pragma unroll
      for (int t = 0; t < ND; ++t) {
        const bf16* vrow = &Vb[(t * 32 + lq) * LDV + 16 * u + 4 * lh];
        const bf16x4 lo = *reinterpret_cast<const bf16x4*>(vrow);
        const bf16x4 hi = *reinterpret_cast<const bf16x4*>(vrow + 8);
        bf16x8 vf;
        vf[0] = lo[0]; vf[1] = lo[1]; vf[2] = lo[2]; vf[3] = lo[3];
        vf[4] = hi[0]; vf[5] = hi[1]; vf[6] = hi[2]; vf[7] = hi[3];
#pragma unroll
        for (int g = 0; g < QG; ++g) o[g][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[g], o[g][t], 0, 0, 0);
      }
    }
    if constexpr (FULL && PF2) {
      // The next tile's data was fetched a tile ago; of the loads issued
      // since (this tile's fetch), the ones every lane issues are the last
      // KV / NT + VV / NT in program order, so waiting down to that many
      // leaves only them in flight.
      wait_vmcnt<KV / NT + VV / NT>();
    }
    if (more) stage_any(b ^ 1, k0 + KT, sk, sv);
    __syncthreads();
  };
  const int nfull = a.Nk / KT;
  int it = 0;
  // Every load issued so far (the queries, the first tiles) has landed
  // before the loops start: otherwise the compiler cannot tell, inside the
  // loop, that the query registers are no longer pending and waits for all
  // outstanding loads, the prefetch included, before the first product of
  // every tile.
  wait_vmcnt<0>();
  const bool full_ok = FAST && vvec;
  if constexpr (PF2) {
    // pairs whose fetch targets (tiles it + 2 and it + 3) are both full
    if (full_ok)
      for (; (it + 4) * KT <= a.Nk; it += 2) {
        tile(BC<false>{}, BC<FAST>{}, it * KT, it, rk0, rv0, rk1, rv1, BC<false>{});
        tile(BC<false>{}, BC<FAST>{}, (it + 1) * KT, it + 1, rk1, rv1, rk0, rv0, BC<false>{});
      }
    for (; it + 1 < nfull; it += 2) {
      tile(BC<false>{}, BC<false>{}, it * KT, it, rk0, rv0, rk1, rv1, BC<false>{});
      tile(BC<false>{}, BC<false>{}, (it + 1) * KT, it + 1, rk1, rv1, rk0, rv0, BC<false>{});
    }
    if (it < nfull) {
      tile(BC<false>{}, BC<false>{}, it * KT, it, rk0, rv0, rk1, rv1, BC<false>{});
      ++it;
    }
  } else {
    if (full_ok)
      for (; (it + 2) * KT <= a.Nk; ++it) tile(BC<false>{}, BC<FAST>{}, it * KT, it, rk0, rv0, rk0, rv0, BC<false>{});
    for (; it < nfull; ++it) tile(BC<false>{}, BC<false>{}, it * KT, it, rk0, rv0, rk0, rv0, BC<false>{});
  }
  // (the partial last tile fetches and stages nothing)
  // The half tail is built for the pre-scaled widths of SD-1.5's heads
  // (d = 40, 80, 160: the 77-token cross-attention's 13-key tail); at the
  // other widths the second tail instance made the kernel spill.
  constexpr bool HALF_OK = QS && (D16 == 48 || D16 == 80 || D16 == 160);
  if constexpr (HALF_OK) {
    if (nfull * KT + 32 >= a.Nk && nfull * KT < a.Nk)
      tile(BC<true>{}, BC<false>{}, nfull * KT, it, rk0, rv0, rk1, rv1, BC<true>{});
    else if (nfull * KT < a.Nk)
      tile(BC<true>{}, BC<false>{}, nfull * KT, it, rk0, rv0, rk1, rv1, BC<false>{});
  } else {
    if (nfull * KT < a.Nk) tile(BC<true>{}, BC<false>{}, nfull * KT, it, rk0, rv0, rk1, rv1, BC<false>{});
  }

  // O^T accumulator: lane holds head dims t*32 + 8(r/4) + 4 lh + [0, 4) of
  // its query; each run of 4 is one 8-byte store.
#pragma unroll
  for (int g = 0; g < QG; ++g) {
    float l = l_run[g];
    if constexpr (SF) {  // the ones row d of V^T accumulated the row sum into O^T row d
      l = 0.f;
#pragma unroll
      for (int t = 0; t < ND; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (32 * t + 8 * (r >> 2) + 4 * lh + (r & 3) == d) l = o[g][t][r];
    }
    const float inv = 1.0f / xor32_sum(l);
    const int q = qb + 32 * g + lq;
    if (q < a.Nq) {
      bf16* O = reinterpret_cast<bf16*>(a.o) + (long)img * a.o_img + (long)q * a.o_ld + hd;
#pragma unroll
      for (int t = 0; t < ND; ++t)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const int dd = t * 32 + 8 * rg + 4 * lh;
          if (dd < d) {
            bf16x4 w;
#pragma unroll
            for (int e = 0; e < 4; ++e) w[e] = (bf16)(o[g][t][4 * rg + e] * inv);
            *reinterpret_cast<bf16x4*>(O + dd) = w;
          }
        }
    }
  }
}

template <int DMAX, int KTF>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgs a) {
  __shared__ float Ks[KTF * DMAX];
  __shared__ float Vs[KTF * DMAX];
  const int tid = threadIdx.x;
  const int img = blockIdx.z, head = blockIdx.y;
  const int q = blockIdx.x * 64 + tid;
  const int kvimg = a.kv_index ? a.kv_index[img] : img;
  const int hd = head * a.d, d = a.d;
  const float* Q = reinterpret_cast<const float*>(a.q) + (long)img * a.q_img + hd;
  const float* K = reinterpret_cast<const float*>(a.k) + (long)kvimg * a.k_img + hd;
  const float* V = reinterpret_cast<const float*>(a.v) + (long)kvimg * a.v_img + hd;
  // q_log2: Q holds q * scale * log2(e), so a score is a base-2 exponent
  const bool l2 = a.q_log2 != 0;
  float qv[DMAX], o[DMAX];
#pragma unroll
  for (int i = 0; i < DMAX; ++i) {
    qv[i] = (q < a.Nq && i < d) ? Q[(long)q * a.q_ld + i] : 0.f;
    o[i] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int k0 = 0; k0 < a.Nk; k0 += KTF) {
    __syncthreads();
    const int nk = min(KTF, a.Nk - k0);
    for (int idx = tid; idx < nk * d; idx += 64) {
      const int key = idx / d, i = idx - key * d;
      Ks[key * DMAX + i] = K[(long)(k0 + key) * a.k_ld + i];
      Vs[key * DMAX + i] = V[(long)(k0 + key) * a.v_ld + i];
    }
    __syncthreads();
    for (int key = 0; key < nk; ++key) {
      float sc = 0.f;
#pragma unroll
      for (int i = 0; i < DMAX; ++i)
        if (i < d) sc = fmaf(qv[i], Ks[key * DMAX + i], sc);
      if (!l2) sc *= a.scale;
      const float mn = fmaxf(m, sc);
      const float al = l2 ? exp2f(m - mn) : expf(m - mn), p = l2 ? exp2f(sc - mn) : expf(sc - mn);
      l = l * al + p;
#pragma unroll
      for (int i = 0; i < DMAX; ++i)
        if (i < d) o[i] = o[i] * al + p * Vs[key * DMAX + i];
      m = mn;
    }
  }
  if (q < a.Nq) {
    float* O = reinterpret_cast<float*>(a.o) + (long)img * a.o_img + (long)q * a.o_ld + hd;
#pragma unroll
    for (int i = 0; i < DMAX; ++i)
      if (i < d) O[i] = o[i] / l;
  }
}

template <int D16, bool QS, bool MF, bool SF>
static void launch_d(const AttnArgs& a, hipStream_t s) {
  // Narrow heads take two query groups per wave (half the K/V traffic and
  // fragment reads per query, still two waves per SIMD); wider ones one.
  constexpr int NW = 4, QG = D16 <= 64 ? 2 : 1;
  dim3 grid((a.Nq + 32 * NW * QG - 1) / (32 * NW * QG), a.heads, a.imgs);
  attn_bf16_kernel<D16, QS, MF, SF, NW, QG><<<grid, 64 * NW, 0, s>>>(a);
}

// Head widths d (multiples of 8) whose 16-rounding is D16: d = D16 - 8
// carries the max (with pre-scaled queries) and the sum in the products;
// d = D16 carries the sum when D16 is an odd multiple of 16.
template <int D16>
static void launch_w(const AttnArgs& a, hipStream_t s) {
  constexpr bool odd = (D16 / 16) % 2 == 1;
  if (a.q_log2) {
    if (a.d < D16)
      launch_d<D16, true, true, true>(a, s);
    else
      launch_d<D16, true, false, odd>(a, s);
  } else {
    if (a.d < D16)
      launch_d<D16, false, false, true>(a, s);
    else
      launch_d<D16, false, false, odd>(a, s);
  }
}

bool attention_width_ok(int d) {
  if (d < 8 || d % 8) return false;
  switch ((d + 15) / 16 * 16) {
    case 16: case 32: case 48: case 64: case 80: case 96: case 128: case 160: case 192: case 256: return true;
    default: return false;
  }
}

hipError_t launch_attention(DType dt, const AttnArgs& a, hipStream_t s) {
  if (a.imgs <= 0 || a.Nq <= 0) return hipSuccess;
  if (dt == BF16) {
    if (!attention_width_ok(a.d) || !a.vt) return hipErrorInvalidValue;
    switch ((a.d + 15) / 16 * 16) {
      case 16: launch_w<16>(a, s); break;
      case 32: launch_w<32>(a, s); break;
      case 48: launch_w<48>(a, s); break;
      case 64: launch_w<64>(a, s); break;
      case 80: launch_w<80>(a, s); break;
      case 96: launch_w<96>(a, s); break;
      case 128: launch_w<128>(a, s); break;
      case 160: launch_w<160>(a, s); break;
      case 192: launch_w<192>(a, s); break;
      case 256: launch_w<256>(a, s); break;
      default: return hipErrorInvalidValue;
    }
  } else {
    if (a.vt || a.d <= 0) return hipErrorInvalidValue;
    dim3 grid((a.Nq + 63) / 64, a.heads, a.imgs);
    // (the wide heads keep q and o in scratch: the fp32 path is the
    // reference-precision path for small configurations, not a fast one)
    if (a.d <= 16)
      attn_f32_kernel<16, 64><<<grid, 64, 0, s>>>(a);
    else if (a.d <= 64)
      attn_f32_kernel<64, 64><<<grid, 64, 0, s>>>(a);
    else if (a.d <= 128)
      attn_f32_kernel<128, 32><<<grid, 64, 0, s>>>(a);
    else if (a.d <= 256)
      attn_f32_kernel<256, 16><<<grid, 64, 0, s>>>(a);
    else
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace sd
