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

template <int DP>  // head width padded to a multiple of 32
__global__ __launch_bounds__(256) void attn_bf16_kernel(AttnArgs a) {
  using namespace fa;
  constexpr int LDK = DP + 8, LDV = KT + 8, NJ = DP / 16, ND = DP / 32;
  __shared__ __attribute__((aligned(16))) bf16 Ks[KT * LDK];
  __shared__ __attribute__((aligned(16))) bf16 Vt[DP * LDV];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int img = blockIdx.z, head = blockIdx.y;
  const int q0 = blockIdx.x * 128 + wave * 32;
  const int kvimg = a.kv_index ? a.kv_index[img] : img;
  const int hd = head * a.d;
  const bf16* Q = reinterpret_cast<const bf16*>(a.q) + (long)img * a.q_img + hd;
  const bf16* K = reinterpret_cast<const bf16*>(a.k) + (long)kvimg * a.kv_img + hd;
  const bf16* V = reinterpret_cast<const bf16*>(a.v) + (long)kvimg * a.kv_img + hd;
  const int lq = lane & 31, lh = lane >> 5;

  // Q^T fragments (B operand): query q0 + lq, head dims 16 j + 8 lh + [0, 8).
  bf16x8 qf[NJ];
  {
    const int q = q0 + lq;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int dd = 16 * j + 8 * lh;
      bf16x8 z = {};
      qf[j] = (q < a.Nq && dd < a.d) ? *reinterpret_cast<const bf16x8*>(Q + (long)q * a.q_ld + dd) : z;
    }
  }
  f32x16 o[ND];
#pragma unroll
  for (int t = 0; t < ND; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[t][r] = 0.f;
  float m_run = -1e30f, l_run = 0.f;
  const float sl2 = a.scale * 1.4426950408889634f;

  for (int k0 = 0; k0 < a.Nk; k0 += KT) {
    __syncthreads();
    // Stage K (key-major) and V^T (dim-major) tiles; zero past Nk and d.
    for (int idx = tid; idx < KT * (DP / 8); idx += 256) {
      const int key = idx / (DP / 8), dc = (idx - key * (DP / 8)) * 8;
      bf16x8 kv = {}, vv = {};
      if (k0 + key < a.Nk && dc < a.d) {
        kv = *reinterpret_cast<const bf16x8*>(K + (long)(k0 + key) * a.kv_ld + dc);
        vv = *reinterpret_cast<const bf16x8*>(V + (long)(k0 + key) * a.kv_ld + dc);
      }
      *reinterpret_cast<bf16x8*>(&Ks[key * LDK + dc]) = kv;
#pragma unroll
      for (int i = 0; i < 8; ++i) Vt[(dc + i) * LDV + key] = vv[i];
    }
    __syncthreads();

    // S^T tiles: rows = keys kt*32 + 8(r/4) + 4 lh + r%4, col = query lq.
    f32x16 s[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kt][r] = 0.f;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&Ks[(kt * 32 + lq) * LDK + 16 * j + 8 * lh]);
        s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[j], s[kt], 0, 0, 0);
      }
    }
    float mt = -1e30f;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = k0 + kt * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
        const float x = key < a.Nk ? s[kt][r] * sl2 : -1e30f;
        s[kt][r] = x;
        mt = fmaxf(mt, x);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const float m_new = fmaxf(m_run, mt);
    const float alpha = exp2f(m_run - m_new);
    m_run = m_new;
    float ps = 0.f;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = exp2f(s[kt][r] - m_new);
        s[kt][r] = p;
        ps += p;
      }
    l_run = l_run * alpha + ps;
#pragma unroll
    for (int t = 0; t < ND; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[t][r] *= alpha;

    // O^T += V^T P^T over four 16-key slices.  Slot (lh, i) of slice u is
    // key 16u + 8(i/4) + 4 lh + i%4, i.e. register 8(u%2) + i of S^T tile u/2.
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      bf16x8 pf;
#pragma unroll
      for (int i = 0; i < 8; ++i) pf[i] = (bf16)s[u >> 1][8 * (u & 1) + i];
#pragma unroll
      for (int t = 0; t < ND; ++t) {
        const bf16* vrow = &Vt[(t * 32 + lq) * LDV + 16 * u + 4 * lh];
        const bf16x4 lo = *reinterpret_cast<const bf16x4*>(vrow);
        const bf16x4 hi = *reinterpret_cast<const bf16x4*>(vrow + 8);
        bf16x8 vf;
        vf[0] = lo[0]; vf[1] = lo[1]; vf[2] = lo[2]; vf[3] = lo[3];
        vf[4] = hi[0]; vf[5] = hi[1]; vf[6] = hi[2]; vf[7] = hi[3];
        o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, o[t], 0, 0, 0);
      }
    }
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.0f / l_tot;
  const int q = q0 + lq;
  if (q < a.Nq) {
    bf16* O = reinterpret_cast<bf16*>(a.o) + (long)img * a.o_img + (long)q * a.o_ld + hd;
#pragma unroll
    for (int t = 0; t < ND; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int dd = t * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
        if (dd < a.d) O[dd] = (bf16)(o[t][r] * inv);
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
  const float* K = reinterpret_cast<const float*>(a.k) + (long)kvimg * a.kv_img + hd;
  const float* V = reinterpret_cast<const float*>(a.v) + (long)kvimg * a.kv_img + hd;
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
      Ks[key * DMAX + i] = K[(long)(k0 + key) * a.kv_ld + i];
      Vs[key * DMAX + i] = V[(long)(k0 + key) * a.kv_ld + i];
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

hipError_t launch_attention(DType dt, const AttnArgs& a, hipStream_t s) {
  if (a.imgs <= 0 || a.Nq <= 0) return hipSuccess;
  if (dt == BF16) {
    dim3 grid((a.Nq + 127) / 128, a.heads, a.imgs);
    const int dp = (a.d + 31) / 32 * 32;
    switch (dp) {
      case 32: attn_bf16_kernel<32><<<grid, 256, 0, s>>>(a); break;
      case 64: attn_bf16_kernel<64><<<grid, 256, 0, s>>>(a); break;
      case 96: attn_bf16_kernel<96><<<grid, 256, 0, s>>>(a); break;
      case 128: attn_bf16_kernel<128><<<grid, 256, 0, s>>>(a); break;
      case 160: attn_bf16_kernel<160><<<grid, 256, 0, s>>>(a); break;
      case 192: attn_bf16_kernel<192><<<grid, 256, 0, s>>>(a); break;
      case 256: attn_bf16_kernel<256><<<grid, 256, 0, s>>>(a); break;
      default: return hipErrorInvalidValue;
    }
  } else {
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
