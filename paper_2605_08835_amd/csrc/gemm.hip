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

// Four consecutive output channels n..n+3 of row m (n % 4 == 0, N % 4 == 0).
template <typename T>
__device__ inline void store4(const Epi& e, int m, int n, const float x[4]) {
  if (e.out_f32) {
    *reinterpret_cast<float4*>(reinterpret_cast<float*>(e.out) + (long)m * e.ldo + n) =
        make_float4(x[0], x[1], x[2], x[3]);
  } else {
    bf16x4 o;
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = (bf16)x[i];
    *reinterpret_cast<bf16x4*>(reinterpret_cast<T*>(e.out) + (long)m * e.ldo + n) = o;
  }
}

template <typename T>
__device__ inline void epilogue4(const Epi& e, int m, int n, float x[4]) {
  if (e.bias) {
    const float4 b = *reinterpret_cast<const float4*>(e.bias + n);
    x[0] += b.x; x[1] += b.y; x[2] += b.z; x[3] += b.w;
  }
  if (e.tbias) {
    const float4 b = *reinterpret_cast<const float4*>(e.tbias + (long)(m / e.hw) * e.tb_ld + e.tb_off + n);
    x[0] += b.x; x[1] += b.y; x[2] += b.z; x[3] += b.w;
  }
  if (e.resid) {
    const bf16x4 r = *reinterpret_cast<const bf16x4*>(reinterpret_cast<const T*>(e.resid) + (long)m * e.ldr + n);
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] += (float)r[i];
  }
  store4<T>(e, m, n, x);
}

// ---------------------------------------------------------------- bf16 MFMA
// Block tile BM x BN x 64, 256 threads = WM x WN waves, each wave a
// (BM/WM) x (BN/WN) sub-tile of 32x32 MFMA accumulators.  Double-buffered
// LDS (one barrier per K step) with the next K tile prefetched into
// registers while the current one feeds the MFMAs.  Rows of both tiles are
// padded by 16 bytes so the 16-byte fragment reads of 8 consecutive rows hit
// distinct banks.  Blocks are renumbered so that the tiles sharing one A
// row band run on the same XCD (blocks are dealt round-robin over 8 XCDs).
namespace mf {
constexpr int BK = 64, LDS_LD = BK + 8;
}

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

// FAST: every segment is a stride-1 3x3 or 1x1 layer on an image of the
// output's size, with cin and the source split c0 multiples of BK, so each
// K tile lies in one (segment, tap, source) and the input pixel of row m
// under tap (ky, kx) is m + (ky-1) W + (kx-1): the per-tile addressing is
// uniform and each row keeps only m and a 9-bit mask of in-image taps.
template <int BM, int BN, int WM, int WN, bool AFF, bool FAST>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 2))) void gemm_bf16_kernel(GemmArgs a) {
  using namespace mf;
  constexpr int TM = BM / WM / 32, TN = BN / WN / 32;  // 32x32 tiles per wave
  constexpr int AR = BM / 32, BR = BN / 32;             // 16-byte chunks per thread
  __shared__ __attribute__((aligned(16))) bf16 As[2][BM * LDS_LD];
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][BN * LDS_LD];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int tiles_n = (a.N + BN - 1) / BN;
  int bid = blockIdx.x;
  const int nb = gridDim.x;
  if ((nb & 7) == 0) bid = (bid & 7) * (nb >> 3) + (bid >> 3);
  const int tm = bid / tiles_n, tn = bid - tm * tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;

  const int kc = tid & 7, lrow = tid >> 3;  // loader: chunk kc of rows lrow + 32 j
  RowPos rp[FAST ? 1 : AR];
  int fm[FAST ? AR : 1], fmask[FAST ? AR : 1];
  if constexpr (FAST) {
    const int W = a.seg[0].Wo, H = a.seg[0].Ho, hw = H * W;
#pragma unroll
    for (int j = 0; j < AR; ++j) {
      const int m = m0 + lrow + 32 * j;
      const int p = m % hw, oy = p / W, ox = p - oy * W;
      int mk = 0;
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const int iy = oy + t / 3 - 1, ix = ox + t % 3 - 1;
        if (iy >= 0 && iy < H && ix >= 0 && ix < W) mk |= 1 << t;
      }
      fm[j] = m;
      fmask[j] = m < a.M ? mk : 0;
    }
  } else {
#pragma unroll
    for (int j = 0; j < AR; ++j) rp[j] = decode_row(a.seg[0], m0 + lrow + 32 * j, a.M);
  }
  const bf16* B = reinterpret_cast<const bf16*>(a.B);

  bf16x8 ra[AR], rb[BR];
  auto gload = [&](int kt) {
    const int k = kt * BK + kc * 8;
    const bf16x8 z = {};
    if constexpr (FAST) {
      // uniform per tile: segment, tap, source and channel base
      const int k0 = kt * BK;
      // (fields picked one by one: selecting a whole kernel-argument struct
      // by a runtime condition would copy it to scratch)
      const bool s1 = k0 >= a.seg[0].K;
      const int kk = s1 ? k0 - a.seg[0].K : k0;
      const int gcin = s1 ? a.seg[1].cin : a.seg[0].cin, gks = s1 ? a.seg[1].ks : a.seg[0].ks;
      const int gc0 = s1 ? a.seg[1].c0 : a.seg[0].c0, gc1 = s1 ? a.seg[1].c1 : a.seg[0].c1;
      const void* gs0 = s1 ? a.seg[1].src0 : a.seg[0].src0;
      const void* gs1 = s1 ? a.seg[1].src1 : a.seg[0].src1;
      const int tap = kk / gcin, cb = kk - tap * gcin;
      const int t9 = gks == 3 ? tap : 4;  // a 1x1 tap is the centre of the 3x3 mask
      const int dpix = gks == 3 ? (tap / 3 - 1) * a.seg[0].Wo + (tap % 3 - 1) : 0;
      const bool in0 = cb < gc0;
      const bf16* src = reinterpret_cast<const bf16*>(in0 ? gs0 : gs1);
      const int cs = in0 ? gc0 : gc1, c = (in0 ? cb : cb - gc0) + kc * 8;
      const bool live = k0 < a.K;
#pragma unroll
      for (int j = 0; j < AR; ++j) {
        const bool ok = live && ((fmask[j] >> t9) & 1);
        ra[j] = ok ? *reinterpret_cast<const bf16x8*>(src + (long)(fm[j] + dpix) * cs + c) : z;
      }
    } else if (k < a.seg[0].K) {
      const int tap = k / a.seg[0].cin, c = k - tap * a.seg[0].cin;
#pragma unroll
      for (int j = 0; j < AR; ++j) {
        if (AFF) {
          ra[j] = a_chunk_bf16(a.seg[0], rp[j], tap, c);
        } else {
          const bf16* p = a_chunk_ptr<bf16>(a.seg[0], rp[j], tap, c);
          ra[j] = p ? *reinterpret_cast<const bf16x8*>(p) : z;
        }
      }
    } else if (k < a.K) {
      const int kk = k - a.seg[0].K;
      const int tap = kk / a.seg[1].cin, c = kk - tap * a.seg[1].cin;
#pragma unroll
      for (int j = 0; j < AR; ++j) {
        const bf16* p = a_chunk_ptr<bf16>(a.seg[1], rp[j], tap, c);
        ra[j] = p ? *reinterpret_cast<const bf16x8*>(p) : z;
      }
    } else {
#pragma unroll
      for (int j = 0; j < AR; ++j) ra[j] = z;
    }
#pragma unroll
    for (int j = 0; j < BR; ++j) {
      const int n = n0 + lrow + 32 * j;
      rb[j] = (n < a.N && k < a.K) ? *reinterpret_cast<const bf16x8*>(B + (long)n * a.ldb + k) : z;
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int j = 0; j < AR; ++j) *reinterpret_cast<bf16x8*>(&As[buf][(lrow + 32 * j) * LDS_LD + kc * 8]) = ra[j];
#pragma unroll
    for (int j = 0; j < BR; ++j) *reinterpret_cast<bf16x8*>(&Bs[buf][(lrow + 32 * j) * LDS_LD + kc * 8]) = rb[j];
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = (a.K + BK - 1) / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  const int lr = lane & 31, lk = 8 * (lane >> 5);
  const int arow = wm * (BM / WM) + lr, brow = wn * (BN / WN) + lr;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
    const bf16* Ab = As[cur];
    const bf16* Bb = Bs[cur];
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(&Ab[(arow + i * 32) * LDS_LD + ks * 16 + lk]);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8*>(&Bb[(brow + j * 32) * LDS_LD + ks * 16 + lk]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }

  // The MFMAs compute C^T tiles (weights as the first operand), so element
  // r of lane l is (output channel 8*(r/4) + 4*(l/32) + r%4, pixel l%32):
  // each lane owns runs of 4 consecutive channels of one pixel and stores
  // them with one 8-byte (bf16) or 16-byte (fp32) write.  Tiles are visited
  // with compile-time indices so the accumulators stay in registers.
  const int hq = 4 * (lane >> 5);
  static_for<0, TM>([&](auto I) {
    static_for<0, TN>([&](auto J) {
      const f32x16 v = acc[I.value][J.value];
      const int m = m0 + wm * (BM / WM) + I.value * 32 + lr;
      const int nt = n0 + wn * (BN / WN) + J.value * 32;
      if (m < a.M) {
        if (a.epi.geglu) {
          // packed columns 32t + u (a) and 32t + 16 + u (gate) -> channel 16t + u
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            const int n = nt + 8 * q + hq;
            if (n < a.N) {
              float x[4], g[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                x[e] = v[4 * q + e] + a.epi.bias[n + e];
                g[e] = v[4 * (q + 2) + e] + a.epi.bias[n + 16 + e];
                x[e] *= 0.5f * g[e] * (1.0f + erff(g[e] * 0.70710678118654752f));
              }
              store4<bf16>(a.epi, m, nt / 2 + 8 * q + hq, x);
            }
          }
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int n = nt + 8 * q + hq;
            if (n < a.N) {
              float x[4] = {v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]};
              epilogue4<bf16>(a.epi, m, n, x);
            }
          }
        }
      }
    });
  });
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

static bool fast_seg(const ASeg& g, int Ho, int Wo) {
  return g.stride == 1 && !g.up && (g.ks == 1 || g.ks == 3) && g.Hi == Ho && g.Wi == Wo &&
         g.cin % mf::BK == 0 && (g.c1 == 0 || g.c0 % mf::BK == 0) && g.scale == nullptr;
}

template <int BM, int BN, int WM, int WN>
static void launch_bf16(const GemmArgs& a, hipStream_t s) {
  const long blocks = (long)((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  const ASeg& g0 = a.seg[0];
  const bool fast = fast_seg(g0, g0.Ho, g0.Wo) && (a.seg[1].K == 0 || fast_seg(a.seg[1], g0.Ho, g0.Wo)) &&
                    g0.Ho * g0.Wo > 0;
  if (fast)
    gemm_bf16_kernel<BM, BN, WM, WN, false, true><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(a);
  else if (g0.scale)
    gemm_bf16_kernel<BM, BN, WM, WN, true, false><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(a);
  else
    gemm_bf16_kernel<BM, BN, WM, WN, false, false><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(a);
}

// Tile choice: the widest N tile that divides N (160 covers every SD-1.5 /
// SDXL width: 320, 640, 1280 and their 2x, 3x, 4x, 8x), then the tallest M
// tile that still gives every CU about two blocks.  The choice depends on
// the layer shape and the row count only through M, and no K is split, so a
// row's result never depends on its batch-mates.
hipError_t launch_gemm(DType dt, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (dt == BF16 && (a.N % 4 || a.epi.ldo % 4 || (a.epi.resid && a.epi.ldr % 4) || (a.epi.geglu && a.N % 32)))
    return hipErrorInvalidValue;
  if (dt != BF16 && a.epi.geglu) return hipErrorInvalidValue;
  if (dt == BF16) {
    auto nblk = [&](int bm, int bn) { return (long)((a.M + bm - 1) / bm) * ((a.N + bn - 1) / bn); };
    const long want = 2 * 256;
    if (a.N % 160 == 0) {
      if (nblk(256, 160) >= want)
        launch_bf16<256, 160, 4, 1>(a, s);
      else
        launch_bf16<128, 160, 4, 1>(a, s);
    } else if (a.N % 128 == 0 || a.N > 64) {
      if (nblk(256, 128) >= want)
        launch_bf16<256, 128, 2, 2>(a, s);
      else if (nblk(128, 128) >= want)
        launch_bf16<128, 128, 2, 2>(a, s);
      else
        launch_bf16<64, 128, 2, 2>(a, s);
    } else if (a.N > 32) {
      launch_bf16<128, 64, 4, 1>(a, s);
    } else {
      launch_bf16<256, 32, 4, 1>(a, s);
    }
  } else {
    const long blocks = (long)((a.M + sf::BM - 1) / sf::BM) * ((a.N + sf::BN - 1) / sf::BN);
    gemm_f32_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(a);
  }
  return hipGetLastError();
}

}  // namespace sd
