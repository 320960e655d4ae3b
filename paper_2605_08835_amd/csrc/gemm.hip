// Implicit-GEMM convolution / linear layers.
//
// C[M, N] = A[M, K] * B[K, N] where A is generated on the fly from NHWC
// activations (3x3 / 1x1 taps, stride 2, nearest-2x upsampling, two-source
// channel concat, fused GroupNorm affine + SiLU) and B is the packed weight
// matrix stored N-major with K contiguous.  bf16 runs on MFMA
// (v_mfma_f32_32x32x16_bf16, fp32 accumulation); fp32 runs a SIMT FMA kernel
// (true fp32, no reduced-precision products).
#include "device_common.h"
#include "kernels.h"

namespace sd {

struct RowPos {
  int img, oy, ox;
  bool ok;
};

__device__ inline RowPos decode_row(const ASeg& s, int m, int M) {
  RowPos r;
  r.ok = m < M;
  const int hw = s.Ho * s.Wo;
  const int mm = r.ok ? m : 0;
  r.img = mm / hw;
  const int p = mm - r.img * hw;
  r.oy = p / s.Wo;
  r.ox = p - r.oy * s.Wo;
  return r;
}

// Address of the 8-channel chunk (tap, c) of output pixel r, or null when
// the tap falls into the zero padding.
template <typename T>
__device__ inline const T* a_chunk_ptr(const ASeg& s, const RowPos& r, int tap, int c) {
  int ky = 1, kx = 1;
  if (s.ks == 3) {
    ky = tap / 3;
    kx = tap - ky * 3;
  }
  int iy = r.oy * s.stride + ky - 1, ix = r.ox * s.stride + kx - 1;
  const int Hs = s.up ? 2 * s.Hi : s.Hi, Ws = s.up ? 2 * s.Wi : s.Wi;
  if (!r.ok || iy < 0 || ix < 0 || iy >= Hs || ix >= Ws) return nullptr;
  if (s.up) {
    iy >>= 1;
    ix >>= 1;
  }
  const long pix = ((long)r.img * s.Hi + iy) * s.Wi + ix;
  if (c < s.c0) return reinterpret_cast<const T*>(s.src0) + pix * s.c0 + c;
  return reinterpret_cast<const T*>(s.src1) + pix * s.c1 + (c - s.c0);
}

// 8 transformed A elements as floats (zero in the padding / past K).
template <typename T>
__device__ inline void a_chunk(const ASeg& s, const RowPos& r, int tap, int c, float v[8]) {
  const T* p = a_chunk_ptr<T>(s, r, tap, c);
  if (!p) {
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = 0.f;
    return;
  }
  load8f(p, v);
  if (s.scale) {
    float sc[8], sh[8];
    load8f(s.scale + (long)r.img * s.cin + c, sc);
    load8f(s.shift + (long)r.img * s.cin + c, sh);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      v[i] = v[i] * sc[i] + sh[i];
      if (s.silu) v[i] = silu_f(v[i]);
    }
  }
}

// bf16 chunk: raw 16-byte copy when no transform applies.
__device__ inline bf16x8 a_chunk_bf16(const ASeg& s, const RowPos& r, int tap, int c) {
  bf16x8 z = {};
  const bf16* p = a_chunk_ptr<bf16>(s, r, tap, c);
  if (!p) return z;
  bf16x8 v = *reinterpret_cast<const bf16x8*>(p);
  if (s.scale) {
    float sc[8], sh[8];
    load8f(s.scale + (long)r.img * s.cin + c, sc);
    load8f(s.shift + (long)r.img * s.cin + c, sh);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      float f = (float)v[i] * sc[i] + sh[i];
      if (s.silu) f = silu_f(f);
      v[i] = (bf16)f;
    }
  }
  return v;
}

template <typename T>
__device__ inline void epilogue_store(const Epi& e, int row, int col, float v) {
  if (e.bias) v += e.bias[col];
  if (e.tbias) v += e.tbias[(long)(row / e.hw) * e.tb_ld + e.tb_off + col];
  if (e.resid) v += to_f(reinterpret_cast<const T*>(e.resid)[(long)row * e.ldr + col]);
  if (e.out_f32)
    reinterpret_cast<float*>(e.out)[(long)row * e.ldo + col] = v;
  else
    reinterpret_cast<T*>(e.out)[(long)row * e.ldo + col] = from_f<T>(v);
}

// ---------------------------------------------------------------- bf16 MFMA
namespace mf {
constexpr int BM = 128, BN = 128, BK = 64, LDS_LD = BK + 8;
}

__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmArgs a) {
  using namespace mf;
  __shared__ __attribute__((aligned(16))) bf16 As[BM * LDS_LD];
  __shared__ __attribute__((aligned(16))) bf16 Bs[BN * LDS_LD];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int tiles_n = (a.N + BN - 1) / BN;
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x - tm * tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;

  const int kc = tid & 7, lrow = tid >> 3;  // loader: chunk kc of rows lrow + 32 j
  RowPos rp[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) rp[j] = decode_row(a.seg[0], m0 + lrow + 32 * j, a.M);
  const bf16* B = reinterpret_cast<const bf16*>(a.B);

  bf16x8 ra[4], rb[4];
  auto gload = [&](int kt) {
    const int k = kt * BK + kc * 8;
    const bf16x8 z = {};
    if (k < a.seg[0].K) {
      const int tap = k / a.seg[0].cin, c = k - tap * a.seg[0].cin;
#pragma unroll
      for (int j = 0; j < 4; ++j) ra[j] = a_chunk_bf16(a.seg[0], rp[j], tap, c);
    } else if (k < a.K) {
      const int kk = k - a.seg[0].K;
      const int tap = kk / a.seg[1].cin, c = kk - tap * a.seg[1].cin;
#pragma unroll
      for (int j = 0; j < 4; ++j) ra[j] = a_chunk_bf16(a.seg[1], rp[j], tap, c);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) ra[j] = z;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + lrow + 32 * j;
      rb[j] = (n < a.N && k < a.K) ? *reinterpret_cast<const bf16x8*>(B + (long)n * a.ldb + k) : z;
    }
  };
  auto sstore = [&]() {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      *reinterpret_cast<bf16x8*>(&As[(lrow + 32 * j) * LDS_LD + kc * 8]) = ra[j];
      *reinterpret_cast<bf16x8*>(&Bs[(lrow + 32 * j) * LDS_LD + kc * 8]) = rb[j];
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = (a.K + BK - 1) / BK;
  gload(0);
  sstore();
  __syncthreads();
  const int lr = lane & 31, lk = 8 * (lane >> 5);
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 af[2], bfr[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(&As[(wm * 64 + i * 32 + lr) * LDS_LD + ks * 16 + lk]);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8*>(&Bs[(wn * 64 + j * 32 + lr) * LDS_LD + ks * 16 + lk]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
    if (kt + 1 < nk) {
      sstore();
      __syncthreads();
    }
  }

  // Accumulator layout of a 32x32 tile: element r of lane l is
  // (row 8*(r/4) + 4*(l/32) + r%4, col l%32).
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int col = n0 + wn * 64 + j * 32 + lr;
        if (row < a.M && col < a.N) epilogue_store<bf16>(a.epi, row, col, acc[i][j][r]);
      }
}

// ---------------------------------------------------------------- fp32 SIMT
namespace sf {
constexpr int BM = 64, BN = 64, BK = 16;
}

__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a) {
  using namespace sf;
  __shared__ float As[BK][BM + 4];
  __shared__ float Bs[BK][BN + 4];
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  const int tiles_n = (a.N + BN - 1) / BN;
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x - tm * tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  const bool loads_a = tid < 128;
  const int lrow = (tid & 127) >> 1, kc = tid & 1;
  const RowPos rp = decode_row(a.seg[0], m0 + lrow, a.M);
  const float* B = reinterpret_cast<const float*>(a.B);

  float acc[4][4] = {};
  const int nk = (a.K + BK - 1) / BK;
  for (int kt = 0; kt < nk; ++kt) {
    const int k = kt * BK + kc * 8;
    float v[8];
    if (loads_a) {
      if (k < a.seg[0].K) {
        const int tap = k / a.seg[0].cin, c = k - tap * a.seg[0].cin;
        a_chunk<float>(a.seg[0], rp, tap, c, v);
      } else if (k < a.K) {
        const int kk = k - a.seg[0].K;
        const int tap = kk / a.seg[1].cin, c = kk - tap * a.seg[1].cin;
        a_chunk<float>(a.seg[1], rp, tap, c, v);
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = 0.f;
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) As[kc * 8 + i][lrow] = v[i];
    } else {
      const int n = n0 + lrow;
      if (n < a.N && k < a.K) {
        load8f(B + (long)n * a.ldb + k, v);
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = 0.f;
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) Bs[kc * 8 + i][lrow] = v[i];
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = m0 + ty * 4 + i, col = n0 + tx * 4 + j;
      if (row < a.M && col < a.N) epilogue_store<float>(a.epi, row, col, acc[i][j]);
    }
}

hipError_t launch_gemm(DType dt, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (dt == BF16) {
    const long blocks = (long)((a.M + mf::BM - 1) / mf::BM) * ((a.N + mf::BN - 1) / mf::BN);
    gemm_bf16_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(a);
  } else {
    const long blocks = (long)((a.M + sf::BM - 1) / sf::BM) * ((a.N + sf::BN - 1) / sf::BN);
    gemm_f32_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(a);
  }
  return hipGetLastError();
}

}  // namespace sd
