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
// LDS with the same permutation.  exp runs as exp2 on pre-scaled scores.
// fp32: one thread per query, K/V tiles in LDS, fp32 online softmax.
#include "device_common.h"
#include "kernels.h"

namespace sd {

namespace fa {
constexpr int KT = 64;  // keys per tile
}

__device__ inline bf16x8 ld16(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }

// D16: head width rounded up to 16 (the QK^T reduction); DP: rounded up to
// 32 (the PV output rows).  QG: groups of 32 queries per wave (the K and V
// fragments read from LDS are reused across the groups).  VT: V is stored
// transposed per image ([channel][token], written so by the projection
// GEMM), so a V^T tile is staged with 16-byte loads and stores.
template <int D16, int QG, bool VT, int NW>
__global__ __launch_bounds__(64 * NW) void attn_bf16_kernel(AttnArgs a) {
  using namespace fa;
  constexpr int NJ = D16 / 16, DP = (D16 + 31) / 32 * 32, ND = DP / 32;
  constexpr int LDK = D16 + 8, LDV = KT + 8, NT = 64 * NW;
  constexpr int KCH = KT * (D16 / 8), VCH = VT ? DP * (KT / 8) : KT * (DP / 8);  // 16-byte chunks per tile
  constexpr int KPT = (KCH + NT - 1) / NT, VPT = (VCH + NT - 1) / NT;           // ... per thread
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
  const bf16* V = reinterpret_cast<const bf16*>(a.v) + (long)kvimg * a.v_img + (VT ? (long)hd * a.v_ld : hd);
  const int lq = lane & 31, lh = lane >> 5;

  // Q^T fragments (B operand): query qb + 32 g + lq, head dims 16 j + 8 lh + [0, 8).
  bf16x8 qf[QG][NJ];
#pragma unroll
  for (int g = 0; g < QG; ++g) {
    const int q = qb + 32 * g + lq;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int dd = 16 * j + 8 * lh;
      const bf16x8 z = {};
      qf[g][j] = (q < a.Nq && dd < a.d) ? ld16(Q + (long)q * a.q_ld + dd) : z;
    }
  }
  f32x16 o[QG][ND];
  float m_run[QG], l_run[QG];
#pragma unroll
  for (int g = 0; g < QG; ++g) {
    m_run[g] = -1e30f;
    l_run[g] = 0.f;
#pragma unroll
    for (int t = 0; t < ND; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[g][t][r] = 0.f;
  }
  const float sl2 = a.scale * 1.4426950408889634f;
  const bool vvec = (a.v_ld & 7) == 0;

  bf16x8 rk[KPT], rv[VPT];
  auto fetch = [&](int k0) {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int idx = tid + NT * i;
      const int key = idx / (D16 / 8), dc = (idx - key * (D16 / 8)) * 8;
      const bf16x8 z = {};
      rk[i] = (idx < KCH && k0 + key < a.Nk && dc < a.d) ? ld16(K + (long)(k0 + key) * a.k_ld + dc) : z;
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int idx = tid + NT * i;
      bf16x8 v = {};
      if constexpr (VT) {
        const int dd = idx / (KT / 8), kc = (idx - dd * (KT / 8)) * 8;
        const int k = k0 + kc;
        if (idx < VCH && dd < a.d && k < a.Nk) {
          const bf16* src = V + (long)dd * a.v_ld + k;
          if (vvec && k + 8 <= a.Nk) {
            v = ld16(src);
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
              if (k + e < a.Nk) v[e] = src[e];
          }
        }
      } else {
        const int key = idx / (DP / 8), dc = (idx - key * (DP / 8)) * 8;
        if (idx < VCH && k0 + key < a.Nk && dc < a.d) v = ld16(V + (long)(k0 + key) * a.v_ld + dc);
      }
      rv[i] = v;
    }
  };
  auto stage = [&](int b) {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int idx = tid + NT * i;
      const int key = idx / (D16 / 8), dc = (idx - key * (D16 / 8)) * 8;
      if (idx < KCH) *reinterpret_cast<bf16x8*>(&Ks[b][key * LDK + dc]) = rk[i];
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int idx = tid + NT * i;
      if (idx >= VCH) continue;
      if constexpr (VT) {
        const int dd = idx / (KT / 8), kc = (idx - dd * (KT / 8)) * 8;
        *reinterpret_cast<bf16x8*>(&Vt[b][dd * LDV + kc]) = rv[i];
      } else {
        const int key = idx / (DP / 8), dc = (idx - key * (DP / 8)) * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) Vt[b][(dc + e) * LDV + key] = rv[i][e];
      }
    }
  };

  fetch(0);
  stage(0);
  __syncthreads();
  for (int k0 = 0, it = 0; k0 < a.Nk; k0 += KT, ++it) {
    const int b = it & 1;
    const bool more = k0 + KT < a.Nk;
    if (more) fetch(k0 + KT);
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
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const bf16x8 kf = ld16(&Kb[(kt * 32 + lq) * LDK + 16 * j + 8 * lh]);
#pragma unroll
        for (int g = 0; g < QG; ++g) s[g][kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[g][j], s[g][kt], 0, 0, 0);
      }
    const bool tail = k0 + KT > a.Nk;
#pragma unroll
    for (int g = 0; g < QG; ++g) {
      if (tail) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (k0 + kt * 32 + 8 * (r >> 2) + 4 * lh + (r & 3) >= a.Nk) s[g][kt][r] = -1e30f;
      }
      float mt = -1e30f;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) mt = fmaxf(mt, s[g][kt][r]);
      mt = fmaxf(mt, __shfl_xor(mt, 32, 64)) * sl2;
      const float m_new = fmaxf(m_run[g], mt);
      const float alpha = __builtin_amdgcn_exp2f(m_run[g] - m_new);
      m_run[g] = m_new;
      float ps = 0.f;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = __builtin_amdgcn_exp2f(fmaf(s[g][kt][r], sl2, -m_new));
          s[g][kt][r] = p;
          ps += p;
        }
      l_run[g] = l_run[g] * alpha + ps;
#pragma unroll
      for (int t = 0; t < ND; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[g][t][r] *= alpha;
    }

    // O^T += V^T P^T over four 16-key slices.  Slot (lh, i) of slice u is
    // key 16u + 8(i/4) + 4 lh + i%4, i.e. register 8(u%2) + i of S^T tile u/2.
#pragma unroll
    for (int u = 0; u < 4; ++u) {
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
    if (more) stage(b ^ 1);
    __syncthreads();
  }

  // O^T accumulator: lane holds head dims t*32 + 8(r/4) + 4 lh + [0, 4) of
  // its query; each run of 4 is one 8-byte store.
#pragma unroll
  for (int g = 0; g < QG; ++g) {
    const float inv = 1.0f / (l_run[g] + __shfl_xor(l_run[g], 32, 64));
    const int q = qb + 32 * g + lq;
    if (q < a.Nq) {
      bf16* O = reinterpret_cast<bf16*>(a.o) + (long)img * a.o_img + (long)q * a.o_ld + hd;
#pragma unroll
      for (int t = 0; t < ND; ++t)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const int dd = t * 32 + 8 * rg + 4 * lh;
          if (dd < a.d) {
            bf16x4 w;
#pragma unroll
            for (int e = 0; e < 4; ++e) w[e] = (bf16)(o[g][t][4 * rg + e] * inv);
            *reinterpret_cast<bf16x4*>(O + dd) = w;
          }
        }
    }
  }
}

template <int DMAX>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgs a) {
  constexpr int KT = 64;
  __shared__ float Ks[KT * DMAX];
  __shared__ float Vs[KT * DMAX];
  const int tid = threadIdx.x;
  const int img = blockIdx.z, head = blockIdx.y;
  const int q = blockIdx.x * 64 + tid;
  const int kvimg = a.kv_index ? a.kv_index[img] : img;
  const int hd = head * a.d, d = a.d;
  const float* Q = reinterpret_cast<const float*>(a.q) + (long)img * a.q_img + hd;
  const float* K = reinterpret_cast<const float*>(a.k) + (long)kvimg * a.k_img + hd;
  const float* V = reinterpret_cast<const float*>(a.v) + (long)kvimg * a.v_img + hd;
  float qv[DMAX], o[DMAX];
#pragma unroll
  for (int i = 0; i < DMAX; ++i) {
    qv[i] = (q < a.Nq && i < d) ? Q[(long)q * a.q_ld + i] : 0.f;
    o[i] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int k0 = 0; k0 < a.Nk; k0 += KT) {
    __syncthreads();
    const int nk = min(KT, a.Nk - k0);
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
      sc *= a.scale;
      const float mn = fmaxf(m, sc);
      const float al = expf(m - mn), p = expf(sc - mn);
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

template <int D16, int QG>
static void launch_d(const AttnArgs& a, hipStream_t s) {
  constexpr int NW = 4;
  dim3 grid((a.Nq + 32 * NW * QG - 1) / (32 * NW * QG), a.heads, a.imgs);
  if (a.vt)
    attn_bf16_kernel<D16, QG, true, NW><<<grid, 64 * NW, 0, s>>>(a);
  else
    attn_bf16_kernel<D16, QG, false, NW><<<grid, 64 * NW, 0, s>>>(a);
}

hipError_t launch_attention(DType dt, const AttnArgs& a, hipStream_t s) {
  if (a.imgs <= 0 || a.Nq <= 0) return hipSuccess;
  if (dt == BF16) {
    switch ((a.d + 15) / 16 * 16) {
      case 16: launch_d<16, 1>(a, s); break;
      case 32: launch_d<32, 1>(a, s); break;
      case 48: launch_d<48, 1>(a, s); break;
      case 64: launch_d<64, 1>(a, s); break;
      case 80: launch_d<80, 1>(a, s); break;
      case 96: launch_d<96, 1>(a, s); break;
      case 128: launch_d<128, 1>(a, s); break;
      case 160: launch_d<160, 1>(a, s); break;
      case 192: launch_d<192, 1>(a, s); break;
      case 256: launch_d<256, 1>(a, s); break;
      default: return hipErrorInvalidValue;
    }
  } else {
    if (a.vt) return hipErrorInvalidValue;
    dim3 grid((a.Nq + 63) / 64, a.heads, a.imgs);
    if (a.d <= 16)
      attn_f32_kernel<16><<<grid, 64, 0, s>>>(a);
    else if (a.d <= 64)
      attn_f32_kernel<64><<<grid, 64, 0, s>>>(a);
    else
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace sd
