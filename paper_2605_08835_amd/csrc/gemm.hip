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
  if (col < e.qcols) v *= e.qscale;
  if (e.out_f32)
    reinterpret_cast<float*>(e.out)[(long)row * e.ldo + col] = v;
  else
    reinterpret_cast<T*>(e.out)[(long)row * e.ldo + col] = from_f<T>(v);
}

// Output row of GEMM row m (the upsample phases write every other pixel of
// every other image row).
__device__ inline long out_row(const Epi& e, int m) {
  if (!e.phase) return m;
  const int hw = e.ph_h * e.ph_w, img = m / hw, p = m - img * hw, y = p / e.ph_w, x = p - y * e.ph_w;
  const int py = (e.phase - 1) >> 1, px = (e.phase - 1) & 1;
  return (long)img * 4 * hw + (long)(2 * y + py) * (2 * e.ph_w) + 2 * x + px;
}

// Four consecutive output channels n..n+3 of row m (n % 4 == 0, N % 4 == 0).
template <typename T>
__device__ inline void store4(const Epi& e, int m, int n, const float x[4]) {
  const long r = out_row(e, m);
  if (e.out_f32) {
    *reinterpret_cast<float4*>(reinterpret_cast<float*>(e.out) + r * e.ldo + n) =
        make_float4(x[0], x[1], x[2], x[3]);
  } else {
    bf16x4 o;
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = (bf16)x[i];
    *reinterpret_cast<bf16x4*>(reinterpret_cast<T*>(e.out) + r * e.ldo + n) = o;
  }
}

// Row scale (a folded LayerNorm's rstd); rows at or past M read nothing.
__device__ inline float row_scale(const Epi& e, int m, int M) {
  return (e.rowscale && m < M) ? e.rowscale[m] : 1.0f;
}

template <typename T>
__device__ inline void epilogue4(const Epi& e, int m, int n, float x[4]) {
  if (e.rowscale) {
    const float rs = e.rowscale[m];
    x[0] *= rs; x[1] *= rs; x[2] *= rs; x[3] *= rs;
  }
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
  if (n < e.qcols) {
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] *= e.qscale;
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

// The MFMAs compute C^T tiles (weights as the first operand), so element r
// of lane l is (output channel 8*(r/4) + 4*(l/32) + r%4, pixel l%32): each
// lane owns runs of 4 consecutive channels of one pixel and stores them with
// one 8-byte (bf16) or 16-byte (fp32) write.  Tiles are visited with
// compile-time indices so the accumulators stay in registers.
template <int BM, int BN, int WM, int WN, int TM, int TN>
__device__ __forceinline__ void epilogue_tiles(const GemmArgs& a, const f32x16 (&acc)[TM][TN], int m0, int n0,
                                               int wm, int wn, int lane) {
  const int lr = lane & 31, hq = 4 * (lane >> 5);
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
              const float rs = row_scale(a.epi, m, a.M);
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                x[e] = fmaf(v[4 * q + e], rs, a.epi.bias[n + e]);
                g[e] = fmaf(v[4 * (q + 2) + e], rs, a.epi.bias[n + 16 + e]);
                x[e] *= gelu_as(g[e]);
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
              if (a.epi.vt_out && n >= a.epi.vt_col0) {
                // transposed store: lanes l and l+1 hold consecutive tokens
                const float rs = row_scale(a.epi, m, a.M);
#pragma unroll
                for (int e = 0; e < 4; ++e) x[e] *= rs;
                const int img = m / a.epi.vt_hw, tok = m - img * a.epi.vt_hw;
                bf16* o = reinterpret_cast<bf16*>(a.epi.vt_out) + (long)img * a.epi.vt_img +
                          (long)(n - a.epi.vt_col0) * a.epi.vt_ld + tok;
#pragma unroll
                for (int e = 0; e < 4; ++e) o[(long)e * a.epi.vt_ld] = (bf16)x[e];
              } else {
                epilogue4<bf16>(a.epi, m, n, x);
              }
            }
          }
        }
      }
    });
  });
}

// Epilogue through LDS for bf16 outputs with no transposed part: each wave
// finishes its values in registers (bias, time bias, GEGLU, residual, query
// scale), writes 32 rows of its tile as bf16 into a private LDS region, then
// stores them back row-contiguous, 16 bytes per lane, so a wave writes whole
// runs instead of 32 scattered 8-byte pieces.  A residual is first copied
// into the same region row-contiguous, and each lane picks up its own
// elements there before overwriting them with the result (one rounding).
// Row stride of the region: the wave's columns plus 8 (16 bytes), which
// keeps rows 16-byte aligned and the 8-byte writes of 32 consecutive rows at
// most two to a bank.
template <int OW>
constexpr int STAGED_LD = OW + 8;

template <int BM, int BN, int WM, int WN, int TM, int TN>
__device__ __forceinline__ void epilogue_staged(const GemmArgs& a, const f32x16 (&acc)[TM][TN], int m0, int n0,
                                                int wm, int wn, int lane, bf16* R) {
  constexpr int WC = BN / WN;  // the wave's accumulator columns
  constexpr int LD = STAGED_LD<WC>;
  const Epi& e = a.epi;
  const bool geglu = e.geglu;
  const int OW = geglu ? WC / 2 : WC;  // output columns of the wave
  const int ncol0 = (geglu ? n0 / 2 : n0) + wn * OW;
  const int lr = lane & 31, hq = 4 * (lane >> 5);
  const bf16* resid = reinterpret_cast<const bf16*>(e.resid);
  // Residual rows (never with GEGLU, so a row has WC / 8 chunks): every load
  // of a 32-row group is issued before the first is used, and the next
  // group's loads are in flight while this group is stored, so the epilogue
  // waits for memory about once instead of once per chunk.
  constexpr int RCH = WC / 8, RPL = 32 * RCH / 64;
  static_assert((32 * RCH) % 64 == 0, "residual chunks spread evenly over the lanes");
  bf16x8 rres[RPL];
  auto load_resid = [&](int mrow0) {
#pragma unroll
    for (int u = 0; u < RPL; ++u) {
      const int c = lane + 64 * u, row = c / RCH, ch = c - row * RCH;
      const int m = mrow0 + row;
      bf16x8 r = {};
      if (m < a.M) r = *reinterpret_cast<const bf16x8*>(resid + (long)m * e.ldr + ncol0 + ch * 8);
      rres[u] = r;
    }
  };
  if (resid) load_resid(m0 + wm * (BM / WM));
  // The bias of the columns the lane finishes in 32-column tile J (columns
  // nt + 8 q + hq + [0, 4); with GEGLU q = 0, 1 are the value and q = 2, 3
  // the gate columns), loaded one tile ahead of its use.
  auto load_bias = [&](int J, float4 (&b)[4]) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      b[q] = e.bias ? *reinterpret_cast<const float4*>(e.bias + n0 + wn * WC + J * 32 + 8 * q + hq)
                    : make_float4(0.f, 0.f, 0.f, 0.f);
  };
  static_for<0, TM>([&](auto I) {
    const int mrow0 = m0 + wm * (BM / WM) + I.value * 32;
    if (resid) {  // (not with GEGLU)
#pragma unroll
      for (int u = 0; u < RPL; ++u) {
        const int c = lane + 64 * u, row = c / RCH, ch = c - row * RCH;
        *reinterpret_cast<bf16x8*>(R + row * LD + ch * 8) = rres[u];
      }
      asm volatile("" ::: "memory");  // (one wave's LDS accesses complete in order)
    }
    static_for<0, TN>([&](auto J) {
      float4 bj[4];
      load_bias(J.value, bj);
      const f32x16 v = acc[I.value][J.value];
      const int nt = n0 + wn * WC + J.value * 32;
      const int m = mrow0 + lr;
      const float rs = row_scale(e, m, a.M);
      if (geglu) {
        // packed columns 32t + u (a) and 32t + 16 + u (gate) -> channel 16t + u
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const float ba[4] = {bj[q].x, bj[q].y, bj[q].z, bj[q].w};
          const float bg[4] = {bj[q + 2].x, bj[q + 2].y, bj[q + 2].z, bj[q + 2].w};
          float x[4];
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const float av = fmaf(v[4 * q + k], rs, ba[k]);
            const float g = fmaf(v[4 * (q + 2) + k], rs, bg[k]);
            x[k] = av * gelu_as(g);
          }
          bf16x4 o;
#pragma unroll
          for (int k = 0; k < 4; ++k) o[k] = (bf16)x[k];
          *reinterpret_cast<bf16x4*>(R + lr * LD + J.value * 16 + 8 * q + hq) = o;
        }
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int n = nt + 8 * q + hq;
          // (one rounding for scale and bias, written out so that it does not
          // depend on the compiler's contraction choices; bj is 0 without a bias)
          float x[4] = {fmaf(v[4 * q], rs, bj[q].x), fmaf(v[4 * q + 1], rs, bj[q].y),
                        fmaf(v[4 * q + 2], rs, bj[q].z), fmaf(v[4 * q + 3], rs, bj[q].w)};
          if (e.tbias && m < a.M) {
            const float4 b = *reinterpret_cast<const float4*>(e.tbias + (long)(m / e.hw) * e.tb_ld + e.tb_off + n);
            x[0] += b.x; x[1] += b.y; x[2] += b.z; x[3] += b.w;
          }
          bf16* slot = R + lr * LD + J.value * 32 + 8 * q + hq;
          if (resid) {
            const bf16x4 r = *reinterpret_cast<const bf16x4*>(slot);
#pragma unroll
            for (int k = 0; k < 4; ++k) x[k] += (float)r[k];
          }
          if (n < e.qcols) {
#pragma unroll
            for (int k = 0; k < 4; ++k) x[k] *= e.qscale;
          }
          bf16x4 o;
#pragma unroll
          for (int k = 0; k < 4; ++k) o[k] = (bf16)x[k];
          *reinterpret_cast<bf16x4*>(slot) = o;
        }
      }
    });
    asm volatile("" ::: "memory");
    if (resid && I.value + 1 < TM) load_resid(mrow0 + 32);
    // Every LDS read of a run of chunks is issued before its first store,
    // so the stores wait for the LDS once per run rather than once per
    // chunk; the row width in chunks is a compile-time constant per case.
    auto store_rows = [&](auto cpc) {
      constexpr int CP = decltype(cpc)::value, NCH = 32 * CP / 64, SH = (NCH + 1) / 2;
      static_assert((32 * CP) % 64 == 0, "row chunks spread evenly over the lanes");
      const int nout = geglu ? a.N / 2 : a.N;
#pragma unroll
      for (int h = 0; h < NCH; h += SH) {
        bf16x8 ob[SH];
#pragma unroll
        for (int u = 0; u < SH; ++u) {
          if (h + u < NCH) {
            const int c = lane + 64 * (h + u), row = c / CP, ch = c - row * CP;
            ob[u] = *reinterpret_cast<const bf16x8*>(R + row * LD + ch * 8);
          }
        }
#pragma unroll
        for (int u = 0; u < SH; ++u) {
          if (h + u < NCH) {
            const int c = lane + 64 * (h + u), row = c / CP, ch = c - row * CP;
            const int m = mrow0 + row;
            if (m < a.M && ncol0 + ch * 8 < nout)
              *reinterpret_cast<bf16x8*>(reinterpret_cast<bf16*>(e.out) + out_row(e, m) * e.ldo + ncol0 + ch * 8) =
                  ob[u];
          }
        }
      }
    };
    if (geglu)
      store_rows(IC<WC / 16>{});
    else
      store_rows(IC<WC / 8>{});
    asm volatile("" ::: "memory");
  });
}

// Epilogue of the large wave tiles (128 x 128 per wave, accumulators in
// AGPRs): each 32-row group of the wave is first written raw (fp32) into a
// wave-private LDS slab, then finished from there in row-contiguous runs of
// 8 outputs per lane (bias, time bias, residual), with the same arithmetic
// as the other epilogues.  Reading the accumulators only to copy them keeps
// the register demand low (the register-staged epilogue spilled here).
// The host sends only layers without GEGLU, a row scale, query columns, a
// transposed part or an fp32 output.
template <int WC>
constexpr int SLAB_LD = WC + 4;  // floats per slab row

template <int BM, int BN, int WM, int WN, int TM, int TN>
__device__ __forceinline__ void epilogue_slab(const GemmArgs& a, const f32x16 (&acc)[TM][TN], int m0, int n0,
                                              int wm, int wn, int lane, float* R) {
  constexpr int WC = BN / WN;
  constexpr int LD = SLAB_LD<WC>;
  constexpr int CP = WC / 8, NCH = 32 * CP / 64;  // 8-output chunks per row; per lane
  static_assert((32 * CP) % 64 == 0, "row chunks spread evenly over the lanes");
  const Epi& e = a.epi;
  const int lr = lane & 31, hq = 4 * (lane >> 5);
  const int nc0 = n0 + wn * WC;  // first column of the wave
  const bf16* resid = reinterpret_cast<const bf16*>(e.resid);
  static_for<0, TM>([&](auto I) {
    const int mrow0 = m0 + wm * (BM / WM) + I.value * 32;
    static_for<0, TN>([&](auto J) {
      const f32x16 v = acc[I.value][J.value];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<float4*>(R + lr * LD + J.value * 32 + 8 * q + hq) =
            make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
    });
    asm volatile("" ::: "memory");  // (one wave's LDS accesses complete in order)
    bf16x8 rr[NCH];
    if (resid) {
#pragma unroll
      for (int u = 0; u < NCH; ++u) {
        const int c = lane + 64 * u, row = c / CP, ch = c - row * CP, m = mrow0 + row;
        bf16x8 r = {};
        if (m < a.M) r = *reinterpret_cast<const bf16x8*>(resid + (long)m * e.ldr + nc0 + ch * 8);
        rr[u] = r;
      }
    }
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      const int c = lane + 64 * u, row = c / CP, ch = c - row * CP, m = mrow0 + row;
      const int n = nc0 + 8 * ch;
      const float* src = R + row * LD + 8 * ch;
      // (one rounding for the bias: fmaf with scale 1, as in the other epilogues)
      float x[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) x[k] = fmaf(src[k], 1.0f, e.bias ? e.bias[n + k] : 0.f);
      if (e.tbias && m < a.M) {
        const float* tb = e.tbias + (long)(m / e.hw) * e.tb_ld + e.tb_off + n;
#pragma unroll
        for (int k = 0; k < 8; ++k) x[k] += tb[k];
      }
      if (resid) {
#pragma unroll
        for (int k = 0; k < 8; ++k) x[k] += (float)rr[u][k];
      }
      bf16x8 o;
#pragma unroll
      for (int k = 0; k < 8; ++k) o[k] = (bf16)x[k];
      if (m < a.M)
        *reinterpret_cast<bf16x8*>(reinterpret_cast<bf16*>(e.out) + out_row(e, m) * e.ldo + n) = o;
    }
    asm volatile("" ::: "memory");
  });
}

// The transposed part of a QKV projection (V written [image][channel][token]
// for the attention kernel): the wave stages its 32 tokens x WC channels
// channel-major, then stores 16-byte runs of 8 consecutive tokens.  Needs
// the 32 tokens in one image at a multiple of 32 (vt_hw % 32 == 0) and
// 16-byte aligned channel rows (vt_ld % 8 == 0).
template <int BM, int BN, int WM, int WN, int TM, int TN>
__device__ __forceinline__ void epilogue_staged_vt(const GemmArgs& a, const f32x16 (&acc)[TM][TN], int m0, int n0,
                                                   int wm, int wn, int lane, bf16* R) {
  constexpr int WC = BN / WN;
  const Epi& e = a.epi;
  const int lr = lane & 31, hq = 4 * (lane >> 5);
  const int c0 = n0 + wn * WC - e.vt_col0;  // first V channel of the wave
  static_for<0, TM>([&](auto I) {
    const int mrow0 = m0 + wm * (BM / WM) + I.value * 32;
    const float rs = row_scale(e, mrow0 + lr, a.M);
    static_for<0, TN>([&](auto J) {
      const f32x16 v = acc[I.value][J.value];
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int k = 0; k < 4; ++k) R[(J.value * 32 + 8 * q + hq + k) * 32 + lr] = (bf16)(v[4 * q + k] * rs);
    });
    asm volatile("" ::: "memory");  // (one wave's LDS accesses complete in order)
    const int img = mrow0 / e.vt_hw, tok0 = mrow0 - img * e.vt_hw;
    bf16* dst = reinterpret_cast<bf16*>(e.vt_out) + (long)img * e.vt_img + (long)c0 * e.vt_ld + tok0;
    for (int c = lane; c < WC * 4; c += 64) {
      const int ch = c >> 2, part = c & 3;
      if (mrow0 + 8 * part < a.M)  // (M is a multiple of vt_hw, hence of 32)
        *reinterpret_cast<bf16x8*>(dst + (long)ch * e.vt_ld + 8 * part) =
            *reinterpret_cast<const bf16x8*>(R + ch * 32 + 8 * part);
    }
    asm volatile("" ::: "memory");
  });
}

// Loader modes.
//  0: per-thread addressing of any layer (incl. the GroupNorm affine on load).
//  1: every segment is a stride-1 3x3 or 1x1 layer on an image of the
//     output's size with cin and the source split c0 multiples of BK, so a
//     K tile lies in one (segment, tap, source) and the input pixel of row m
//     under tap (ky, kx) is m + (ky-1) W + (kx-1): the tile's addressing is
//     uniform and each row keeps only m and a 9-bit mask of in-image taps.
//  2: one stride-2 or upsampling 3x3 segment with cin a multiple of BK:
//     uniform tap per tile, rows keep (image base pixel, oy, ox).
// Modes 1 and 2 read through buffer resources: a masked-off element gets an
// out-of-range offset, which the hardware returns as zero, so the loads are
// branch-free.

template <int BM, int BN, int BK, int WM, int WN, int MODE, int MINB>
__global__ __launch_bounds__(256, MINB) void gemm_bf16_kernel(GemmArgs a) {
  constexpr int LDS_LD = BK + 8;
  constexpr int TM = BM / WM / 32, TN = BN / WN / 32;  // 32x32 tiles per wave
  constexpr int CPR = BK / 8, RPP = 256 / CPR;         // chunks per row, rows per pass
  constexpr int AR = (BM + RPP - 1) / RPP, BR = (BN + RPP - 1) / RPP;  // 16-byte chunks per thread
  static_assert(BM % RPP == 0, "A tile rows must be a multiple of the rows per loader pass");
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

  const int kc = tid % CPR, lrow = tid / CPR;  // loader: chunk kc of rows lrow + RPP j
  constexpr int NR = MODE == 0 ? 1 : AR;
  RowPos rp[MODE == 0 ? AR : 1];
  int ra0[NR], ra1[NR];  // mode 1: (m, tap mask); mode 2: (image base pixel, oy << 16 | ox)
  const int Ho = a.seg[0].Ho, Wo = a.seg[0].Wo, hwo = Ho * Wo;
  if constexpr (MODE == 1) {
#pragma unroll
    for (int j = 0; j < AR; ++j) {
      const int m = m0 + lrow + RPP * j;
      const int p = m % hwo, oy = p / Wo, ox = p - oy * Wo;
      int mk = 0;
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const int iy = oy + t / 3 - 1, ix = ox + t % 3 - 1;
        if (iy >= 0 && iy < Ho && ix >= 0 && ix < Wo) mk |= 1 << t;
      }
      ra0[j] = m;
      ra1[j] = m < a.M ? mk : 0;
    }
  } else if constexpr (MODE == 2) {
#pragma unroll
    for (int j = 0; j < AR; ++j) {
      const int m = m0 + lrow + RPP * j;
      const int img = m / hwo, p = m - img * hwo, oy = p / Wo, ox = p - oy * Wo;
      ra0[j] = img * a.seg[0].Hi * a.seg[0].Wi;
      ra1[j] = m < a.M ? (oy << 16) | ox : -1;
    }
  } else {
#pragma unroll
    for (int j = 0; j < AR; ++j) rp[j] = decode_row(a.seg[0], m0 + lrow + RPP * j, a.M);
  }
  const __amdgpu_buffer_rsrc_t bres = make_rsrc(a.B, (long)a.N * a.ldb * 2);
  int boff[BR];
#pragma unroll
  for (int j = 0; j < BR; ++j) {
    const int n = n0 + lrow + RPP * j;
    boff[j] = (n < a.N && lrow + RPP * j < BN) ? n * a.ldb * 2 : OOB;
  }

  bf16x8 ra[AR], rb[BR];
  // Uniform loader state of the next K tile (modes 1, 2): segment, tap and
  // channel base, advanced by BK per tile without divisions.
  int st_seg = 0, st_tap = 0, st_cb = 0;
  auto gload = [&](int kt) {
    const int k = kt * BK + kc * 8;
    const bf16x8 z = {};
    if constexpr (MODE != 0) {
      // (fields are picked one by one: selecting a whole kernel-argument
      // struct by a runtime condition would copy it to scratch)
      const int k0 = kt * BK;
      const bool s1 = MODE == 1 && st_seg;
      const int gcin = s1 ? a.seg[1].cin : a.seg[0].cin, gks = s1 ? a.seg[1].ks : a.seg[0].ks;
      const int gc0 = s1 ? a.seg[1].c0 : a.seg[0].c0, gc1 = s1 ? a.seg[1].c1 : a.seg[0].c1;
      const void* gs0 = s1 ? a.seg[1].src0 : a.seg[0].src0;
      const void* gs1 = s1 ? a.seg[1].src1 : a.seg[0].src1;
      const int tap = st_tap, cb = st_cb;
      st_cb += BK;
      if (st_cb >= gcin) {
        st_cb = 0;
        if (++st_tap == gks * gks) {
          st_tap = 0;
          st_seg = 1;
        }
      }
      const bool in0 = cb < gc0;
      const int cs = in0 ? gc0 : gc1, c2 = 2 * ((in0 ? cb : cb - gc0) + kc * 8);
      const bool live = k0 < a.K;
      if constexpr (MODE == 1) {
        const long npix = a.M;
        const __amdgpu_buffer_rsrc_t ares = make_rsrc(in0 ? gs0 : gs1, npix * cs * 2);
        // tap offset (dy, dx) and its bit in the 3x3 in-image mask (a 1x1 tap
        // is the centre; an upsample phase's 2x2 taps are four of the nine)
        const int gpy = s1 ? a.seg[1].py : a.seg[0].py, gpx = s1 ? a.seg[1].px : a.seg[0].px;
        const int tdy = gks == 3 ? tap / 3 - 1 : (gks == 2 ? gpy - 1 + (tap >> 1) : 0);
        const int tdx = gks == 3 ? tap % 3 - 1 : (gks == 2 ? gpx - 1 + (tap & 1) : 0);
        const int t9 = (tdy + 1) * 3 + tdx + 1;
        const int dpix = tdy * Wo + tdx;
#pragma unroll
        for (int j = 0; j < AR; ++j) {
          const bool ok = live && ((ra1[j] >> t9) & 1);
          ra[j] = buf_load16(ares, ok ? (ra0[j] + dpix) * cs * 2 + c2 : OOB);
        }
      } else {
        const ASeg& g = a.seg[0];
        const long npix = (long)(a.M / hwo) * g.Hi * g.Wi;
        const __amdgpu_buffer_rsrc_t ares = make_rsrc(in0 ? gs0 : gs1, npix * cs * 2);
        const int ky = tap / 3 - 1, kx = tap % 3 - 1;
#pragma unroll
        for (int j = 0; j < AR; ++j) {
          const int oy = ra1[j] >> 16, ox = ra1[j] & 0xFFFF;
          int iy, ix;
          bool ok;
          if (g.up) {
            iy = oy + ky;
            ix = ox + kx;
            ok = iy >= 0 && iy < 2 * g.Hi && ix >= 0 && ix < 2 * g.Wi;
            iy >>= 1;
            ix >>= 1;
          } else {
            iy = oy * g.stride + ky;
            ix = ox * g.stride + kx;
            ok = iy >= 0 && iy < g.Hi && ix >= 0 && ix < g.Wi;
          }
          ok = ok && live && ra1[j] >= 0;
          ra[j] = buf_load16(ares, ok ? (ra0[j] + iy * g.Wi + ix) * cs * 2 + c2 : OOB);
        }
      }
    } else if (k < a.seg[0].K) {
      const int tap = k / a.seg[0].cin, c = k - tap * a.seg[0].cin;
#pragma unroll
      for (int j = 0; j < AR; ++j) ra[j] = a_chunk_bf16(a.seg[0], rp[j], tap, c);
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
    const bool kin = k < a.K;
#pragma unroll
    for (int j = 0; j < BR; ++j) rb[j] = buf_load16(bres, kin ? boff[j] + 2 * k : OOB);
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int j = 0; j < AR; ++j) *reinterpret_cast<bf16x8*>(&As[buf][(lrow + RPP * j) * LDS_LD + kc * 8]) = ra[j];
#pragma unroll
    for (int j = 0; j < BR; ++j)
      if (BN % RPP == 0 || lrow + RPP * j < BN)
        *reinterpret_cast<bf16x8*>(&Bs[buf][(lrow + RPP * j) * LDS_LD + kc * 8]) = rb[j];
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

  epilogue_tiles<BM, BN, WM, WN>(a, acc, m0, n0, wm, wn, lane);
}




// ------------------------------------------------- bf16 MFMA, direct-to-LDS
// Same tiles and C^T epilogue as above, for the uniform-tap loader modes
// (1, 2), with the operand tiles fetched by buffer_load ... lds: each 64-lane
// load writes 1 KB of LDS contiguously (lane l at byte 16 l), so the loads
// need no registers and three K stages stay in flight.  A tile row holds the
// four 16-byte chunks of a 32-deep K slice; chunk c of row r sits in slot
// c ^ ((r >> 2) & 3), which keeps the fragment reads of 8 consecutive rows
// on distinct banks.  Lane l of a load writes (row 16 i + l / 4, slot l % 4)
// and therefore fetches chunk (l % 4) ^ ((row >> 2) & 3) from global memory.
constexpr int DKS = 32;  // K depth per stage (the split-K and loader-mode granule)

// Slot swizzle of a tile row's 16-byte chunks: the fragment reads of rows
// r..r+15 at one logical chunk land on distinct 16-byte bank groups (4
// chunks per row: 64-byte rows; 8 chunks: 128-byte rows).
template <int CPR>
__device__ __forceinline__ int swz(int r) {
  return CPR == 4 ? (r >> 2) & 3 : (r >> 1) & 7;
}

template <int BM, int BN, int WM, int WN, int MODE, int DNS, int MINB, int DK, bool TI>
__global__ __launch_bounds__(64 * WM * WN, MINB) void gemm_bf16_dma_kernel(GemmArgs a) {
  constexpr int NWV = WM * WN;                          // waves per block
  constexpr int TM = BM / WM / 32, TN = BN / WN / 32;
  constexpr int CPR = DK / 8, RPL = 64 / CPR;           // 16-byte chunks per row, rows per load
  constexpr int AI = BM / RPL, BI = BN / RPL;           // 1 KB loads per tile
  constexpr int AW = AI / NWV, BW = (BI + NWV - 1) / NWV;  // ... per wave (B: some waves one fewer)
  constexpr int LPT_MIN = AW + BI / NWV;                // loads per tile of the lightest wave
  static_assert(DNS >= 2 && DNS <= 4, "pipeline depth");
  static_assert(DK == 32 || DK == 64, "stage depth");
  static_assert(AI % NWV == 0, "A tile must split evenly over the waves");
  // Operand stages (A then B); after the K loop the same LDS stages the
  // output tile for the row-contiguous stores of the epilogue.
  constexpr int OPS = DNS * (BM + BN) * DK, STG = NWV * 32 * STAGED_LD<BN / WN>;
  __shared__ __attribute__((aligned(1024))) bf16 smem[OPS > STG ? OPS : STG];
  bf16* const As = smem;
  bf16* const Bs = smem + DNS * BM * DK;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int tiles_n = (a.N + BN - 1) / BN;
  int bid = blockIdx.x;
  const int nb = gridDim.x;
  if ((nb & 7) == 0) bid = (bid & 7) * (nb >> 3) + (bid >> 3);
  // split-K: blocks split * tiles .. cover K tiles [kb, ke) of their output tile
  const int tiles = (nb / a.ksplit), split = bid / tiles;
  bid -= split * tiles;
  const int tm = bid / tiles_n, tn = bid - tm * tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;

  // Rows and chunks this lane fetches: A load j of this wave is tile load
  // i = wave * AW + j (rows RPL i ..); B load j is i = wave + NWV j.
  const int lrow = lane / CPR, lslot = lane % CPR;
  const int Ho = a.seg[0].Ho, Wo = a.seg[0].Wo, hwo = Ho * Wo;
  int ra0[AW], ra1[AW], achunk[AW];
#pragma unroll
  for (int j = 0; j < AW; ++j) {
    const int r = RPL * (wave * AW + j) + lrow;
    const int m = m0 + r;
    achunk[j] = lslot ^ swz<CPR>(r);
    if constexpr (MODE == 1) {
      const int p = m % hwo, oy = p / Wo, ox = p - oy * Wo;
      int mk = 0;
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const int iy = oy + t / 3 - 1, ix = ox + t % 3 - 1;
        if (iy >= 0 && iy < Ho && ix >= 0 && ix < Wo) mk |= 1 << t;
      }
      ra0[j] = m;
      ra1[j] = m < a.M ? mk : 0;
    } else {
      const int img = m / hwo, p = m - img * hwo, oy = p / Wo, ox = p - oy * Wo;
      ra0[j] = img * a.seg[0].Hi * a.seg[0].Wi;
      ra1[j] = m < a.M ? (oy << 16) | ox : -1;
    }
  }
  const __amdgpu_buffer_rsrc_t bres = make_rsrc(a.B, (long)a.N * a.ldb * 2);
  int boff[BW];
#pragma unroll
  for (int j = 0; j < BW; ++j) {
    const int i = wave + NWV * j;
    const int r = RPL * i + lrow;
    const int n = n0 + r;
    const int c = lslot ^ swz<CPR>(r);
    boff[j] = (i < BI && n < a.N) ? n * a.ldb * 2 + c * 16 : OOB;
  }

  const int nk_all = (a.K + DK - 1) / DK;  // K is a multiple of DK in modes 1, 2
  const int per = (nk_all + a.ksplit - 1) / a.ksplit;
  const int kb = split * per, ke = min(nk_all, kb + per);
  // With TI (images larger than 8x8) the K tiles are visited channel block
  // by channel block, all taps of a block in a row (the packed weights stay
  // tap-major: a tile's weight columns follow from its tap and channel
  // block), so consecutive tiles read the same input rows shifted by a tap
  // and find them in L1 / L2; smaller images (a 256-row tile spans several)
  // go tap by tap.  The order is a property of the layer, like the split.
  constexpr bool tapin = TI;
  int st_seg = 0, st_tap = 0, st_cb = 0;
  {  // loader state at K tile kb
    int kk = kb * DK;
    if (MODE == 1 && kk >= a.seg[0].K) {
      st_seg = 1;
      kk -= a.seg[0].K;
    }
    const int gks = st_seg ? a.seg[1].ks : a.seg[0].ks, gcin = st_seg ? a.seg[1].cin : a.seg[0].cin;
    const int i = kk / DK, taps = gks * gks;
    if constexpr (tapin) {
      st_cb = (i / taps) * DK;
      st_tap = i - (i / taps) * taps;
    } else {
      st_tap = kk / gcin;
      st_cb = kk - st_tap * gcin;
    }
  }
  // The segment fields the refills read, read once as values (selected
  // per tile rather than re-read from the kernel arguments: the scalar
  // loads of a re-read stall the large tiles' loop on their waits).
  const void *g0s0 = a.seg[0].src0, *g0s1 = a.seg[0].src1, *g1s0 = a.seg[1].src0, *g1s1 = a.seg[1].src1;
  const int g0cin = a.seg[0].cin, g0ks = a.seg[0].ks, g0c0 = a.seg[0].c0, g0c1 = a.seg[0].c1, g0py = a.seg[0].py,
            g0px = a.seg[0].px, g0K = a.seg[0].K, gM = a.M;
  const int g1cin = a.seg[1].cin, g1ks = a.seg[1].ks, g1c0 = a.seg[1].c0, g1c1 = a.seg[1].c1, g1py = a.seg[1].py,
            g1px = a.seg[1].px;
  // Issue the loads of K tile kt into stage `stg` (tiles are issued in
  // order).  `live` false: every offset out of range (zeros, no memory
  // access), for the large tiles' refills past the last tile.
  auto issue = [&](int kt, int stg, bool live = true) {
    (void)kt;
    const bool s1 = MODE == 1 && st_seg;
    const int gcin = s1 ? g1cin : g0cin, gks = s1 ? g1ks : g0ks;
    const int gc0 = s1 ? g1c0 : g0c0, gc1 = s1 ? g1c1 : g0c1;
    const void* gs0 = s1 ? g1s0 : g0s0;
    const void* gs1 = s1 ? g1s1 : g0s1;
    const int tap = st_tap, cb = st_cb;
    const int k0 = (s1 ? g0K : 0) + tap * gcin + cb;  // the tile's weight columns
    if constexpr (tapin) {
      if (++st_tap == gks * gks) {
        st_tap = 0;
        st_cb += DK;
        if (st_cb >= gcin) {
          st_cb = 0;
          st_seg = 1;
        }
      }
    } else {
      st_cb += DK;
      if (st_cb >= gcin) {
        st_cb = 0;
        if (++st_tap == gks * gks) {
          st_tap = 0;
          st_seg = 1;
        }
      }
    }
    const bool in0 = cb < gc0;
    const int cs = in0 ? gc0 : gc1, cbase = 2 * (in0 ? cb : cb - gc0);
    bf16* adst = As + stg * BM * DK;
    if constexpr (MODE == 1) {
      const __amdgpu_buffer_rsrc_t ares = make_rsrc(in0 ? gs0 : gs1, (long)gM * cs * 2);
      // tap offset (dy, dx) and its bit in the 3x3 in-image mask (a 1x1 tap
      // is the centre; an upsample phase's 2x2 taps are four of the nine)
      const int gpy = s1 ? g1py : g0py, gpx = s1 ? g1px : g0px;
      // (arithmetic rather than selects, so the refill has no branch: a
      // masked element gets bit 31 set, beyond every source's size)
      const int t3 = tap / 3, is3 = gks == 3, is2 = gks == 2;
      const int tdy = is3 * (t3 - 1) + is2 * (gpy - 1 + (tap >> 1));
      const int tdx = is3 * (tap - 3 * t3 - 1) + is2 * (gpx - 1 + (tap & 1));
      const int t9 = (tdy + 1) * 3 + tdx + 1;
      const int dpix = tdy * Wo + tdx;
      const int dead = (int)!live << 31;
#pragma unroll
      for (int j = 0; j < AW; ++j) {
        const int off = ((ra0[j] + dpix) * cs * 2 + cbase + achunk[j] * 16) | (~(ra1[j] >> t9) << 31) | dead;
        dma16(ares, adst + (wave * AW + j) * 512, off);
      }
    } else {
      const ASeg& g = a.seg[0];
      const long npix = (long)(a.M / hwo) * g.Hi * g.Wi;
      const __amdgpu_buffer_rsrc_t ares = make_rsrc(gs0, npix * cs * 2);
      const int ky = tap / 3 - 1, kx = tap % 3 - 1;
#pragma unroll
      for (int j = 0; j < AW; ++j) {
        const int oy = ra1[j] >> 16, ox = ra1[j] & 0xFFFF;
        int iy, ix;
        bool ok;
        if (g.up) {
          iy = oy + ky;
          ix = ox + kx;
          ok = iy >= 0 && iy < 2 * g.Hi && ix >= 0 && ix < 2 * g.Wi;
          iy >>= 1;
          ix >>= 1;
        } else {
          iy = oy * g.stride + ky;
          ix = ox * g.stride + kx;
          ok = iy >= 0 && iy < g.Hi && ix >= 0 && ix < g.Wi;
        }
        ok = ok && ra1[j] >= 0 && live;
        const int off = ok ? (ra0[j] + iy * g.Wi + ix) * cs * 2 + cbase + achunk[j] * 16 : OOB;
        dma16(ares, adst + (wave * AW + j) * 512, off);
      }
    }
    bf16* bdst = Bs + stg * BN * DK;
#pragma unroll
    for (int j = 0; j < BW; ++j) {
      const int i = wave + NWV * j;
      if (BI % NWV == 0 || i < BI)  // wave-uniform (an OOB row stays beyond the end)
        dma16(bres, bdst + i * 512, (boff[j] + 2 * k0) | ((int)!live << 31));
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = ke - kb;
  const int lr = lane & 31, lh = lane >> 5;
  const int arow = wm * (BM / WM) + lr, brow = wn * (BN / WN) + lr;
  if constexpr (TM * TN > 10) {
    // Large wave tiles run one wave per SIMD, so nothing else hides the
    // K-step barrier or the fragment reads: the loop is software-pipelined.
    // All DNS stages are in flight; the fragments of substep ks + 1 are
    // read before the products of substep ks, and the first fragments of
    // tile kt + 1 (after its wait and the barrier) before the last products
    // of tile kt.  Tile kt + DNS refills the stage of tile kt once every
    // wave has passed that barrier (its reads of tile kt have completed).
    constexpr int KS = DK / 16;
    static_assert(KS % 2 == 0, "fragment sets alternate per substep");
    bf16x8 fa[2][TM], fb[2][TN];
    auto readf = [&](int stg, int ks, bf16x8 (&af)[TM], bf16x8 (&bfr)[TN]) {
      const bf16* Ab = As + stg * BM * DK;
      const bf16* Bb = Bs + stg * BN * DK;
      const int ch = 2 * ks + lh;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = arow + i * 32;
        af[i] = *reinterpret_cast<const bf16x8*>(&Ab[r * DK + 8 * (ch ^ swz<CPR>(r))]);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int r = brow + j * 32;
        bfr[j] = *reinterpret_cast<const bf16x8*>(&Bb[r * DK + 8 * (ch ^ swz<CPR>(r))]);
      }
    };
    // Every stage refill is issued, past the last tile as an all-out-of-range
    // load (zeros into a stage no product reads), so the loop body has no
    // branch and every wait counts the same DNS - 2 tiles in flight.
    static_assert(AI % NWV == 0 && BI % NWV == 0, "every wave issues the same loads");
#pragma unroll
    for (int p = 0; p < DNS; ++p) issue(kb + p, p, p < nk);
    wait_vmcnt<(DNS - 1) * LPT_MIN>();  // tile 0 has landed
    stage_barrier();
    readf(0, 0, fa[0], fb[0]);
    auto products = [&](int cur) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[cur][j], fa[cur][i], acc[i][j], 0, 0, 0);
    };
    // The kernel arguments are loaded here, before the wait below (left to
    // the compiler, some load lazily and are still in flight at the loop;
    // scalar loads return out of order, so every wait for an LDS read in
    // the loop would then wait for all of them).  After it the loop's LDS
    // reads are counted in order: a product waits only for its own
    // fragments.
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const ASeg& sg = a.seg[g];
      asm volatile("" ::"s"(sg.src0), "s"(sg.src1), "s"(sg.cin), "s"(sg.ks), "s"(sg.c0), "s"(sg.c1));
      asm volatile("" ::"s"(sg.K), "s"(sg.py), "s"(sg.px), "s"(sg.Hi), "s"(sg.Wi), "s"(sg.stride), "s"(sg.up));
    }
    {
      const Epi& e = a.epi;
      asm volatile("" ::"s"(e.bias), "s"(e.tbias), "s"(e.tb_ld), "s"(e.tb_off), "s"(e.hw), "s"(e.resid), "s"(e.ldr));
      asm volatile("" ::"s"(e.out), "s"(e.ldo), "s"(e.geglu), "s"(e.qcols), "s"(e.qscale), "s"(e.phase));
      asm volatile("" ::"s"(e.ph_h), "s"(e.ph_w), "s"(e.rowscale), "s"(a.M), "s"(a.N), "s"(e.out_f32));
    }
    wait_lgkm0();
    __builtin_amdgcn_sched_barrier(0);
    // every tile but the last: the last substep reads the next tile
    for (int kt = 0; kt + 1 < nk; ++kt) {
      static_for<0, KS>([&](auto KSI) {
        constexpr int ks = KSI.value, cur = ks & 1, nxt = cur ^ 1;
        if constexpr (ks + 1 < KS) {
          readf(kt % DNS, ks + 1, fa[nxt], fb[nxt]);
          __builtin_amdgcn_sched_barrier(0);  // the reads go out before the products
          products(cur);
        } else {
          __builtin_amdgcn_sched_barrier(0);  // the previous substep's products stay above
          // tiles issued after kt + 1: kt + 2 .. kt + DNS - 1
          wait_vmcnt<(DNS - 2) * LPT_MIN>();
          wait_lgkm0();  // this wave's reads of tile kt are complete
          stage_barrier();
          __builtin_amdgcn_sched_barrier(0);
          readf((kt + 1) % DNS, 0, fa[nxt], fb[nxt]);
          issue(kb + kt + DNS, kt % DNS, kt + DNS < nk);
          products(cur);
          // each fragment read, then each refill load, beside a product
#pragma unroll
          for (int q = 0; q < TM + TN; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
          }
#pragma unroll
          for (int q = 0; q < AW + BW; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
          }
        }
      });
    }
    if (nk > 0) {
      static_for<0, KS>([&](auto KSI) {  // the last tile
        constexpr int ks = KSI.value, cur = ks & 1, nxt = cur ^ 1;
        if constexpr (ks + 1 < KS) readf((nk - 1) % DNS, ks + 1, fa[nxt], fb[nxt]);
        products(cur);
      });
    }
    wait_vmcnt<0>();  // the refills past the last tile have landed
  } else {
#pragma unroll
    for (int p = 0; p < DNS - 1; ++p)
      if (p < nk) issue(kb + p, p);
    for (int kt = 0; kt < nk; ++kt) {
      // Tile kt must have landed; the tiles issued after it may still be in
      // flight (at most DNS-2 of them, fewer near the end of K).
      const int ahead = min(DNS - 2, nk - 1 - kt);
      if (ahead >= 2)
        wait_vmcnt<2 * LPT_MIN>();
      else if (ahead == 1)
        wait_vmcnt<LPT_MIN>();
      else
        wait_vmcnt<0>();
      stage_barrier();
      if (kt + DNS - 1 < nk) issue(kb + kt + DNS - 1, (kt + DNS - 1) % DNS);
      const bf16* Ab = As + (kt % DNS) * BM * DK;
      const bf16* Bb = Bs + (kt % DNS) * BN * DK;
#pragma unroll
      for (int ks = 0; ks < DK / 16; ++ks) {
        const int ch = 2 * ks + lh;
        bf16x8 af[TM], bfr[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int r = arow + i * 32;
          af[i] = *reinterpret_cast<const bf16x8*>(&Ab[r * DK + 8 * (ch ^ swz<CPR>(r))]);
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int r = brow + j * 32;
          bfr[j] = *reinterpret_cast<const bf16x8*>(&Bb[r * DK + 8 * (ch ^ swz<CPR>(r))]);
        }
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
      }
    }
  }
  if (a.ksplit > 1) {
    // raw fp32 partial sums; the reduction kernel applies the epilogue
    const int lr = lane & 31, hq = 4 * (lane >> 5);
    float* P = a.partial + (long)split * a.M * a.N;
    static_for<0, TM>([&](auto I) {
      static_for<0, TN>([&](auto J) {
        const f32x16 v = acc[I.value][J.value];
        const int m = m0 + wm * (BM / WM) + I.value * 32 + lr;
        const int nt = n0 + wn * (BN / WN) + J.value * 32;
        if (m < a.M) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int n = nt + 8 * q + hq;
            if (n < a.N)
              *reinterpret_cast<float4*>(P + (long)m * a.N + n) =
                  make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
          }
        }
      });
    });
    return;
  }
  if constexpr (TM * TN > 10) {
    // large wave tiles: the host sends only layers this epilogue covers
    static_assert(NWV * 32 * SLAB_LD<BN / WN> * 4 <= (int)sizeof(smem), "slabs fit the operand stages");
    __syncthreads();  // every wave is done with the operand stages
    epilogue_slab<BM, BN, WM, WN>(a, acc, m0, n0, wm, wn, lane,
                                  reinterpret_cast<float*>(smem) + wave * 32 * SLAB_LD<BN / WN>);
    return;
  } else {
    static_assert(32 * (BN / WN) <= 32 * STAGED_LD<BN / WN>, "transposed staging fits the region");
    const bool vt_ok = a.epi.vt_out && a.epi.vt_col0 % (BN / WN) == 0 && a.epi.vt_hw % 32 == 0 && a.epi.vt_ld % 8 == 0;
    if ((!a.epi.vt_out || vt_ok) && !a.epi.out_f32 && (!a.epi.resid || !a.epi.geglu)) {
      __syncthreads();  // every wave is done with the operand stages
      bf16* R = smem + wave * 32 * STAGED_LD<BN / WN>;
      if (a.epi.vt_out && n0 + wn * (BN / WN) >= a.epi.vt_col0)
        epilogue_staged_vt<BM, BN, WM, WN>(a, acc, m0, n0, wm, wn, lane, R);
      else
        epilogue_staged<BM, BN, WM, WN>(a, acc, m0, n0, wm, wn, lane, R);
      return;
    }
    epilogue_tiles<BM, BN, WM, WN>(a, acc, m0, n0, wm, wn, lane);
  }
}

// Sum of the split-K partials in split order, then the epilogue.
__global__ void splitk_reduce_kernel(GemmArgs a) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;  // one run of 4 columns
  const int nv = a.N / 4;
  if (i >= (long)a.M * nv) return;
  const int m = (int)(i / nv), n = (int)(i - (long)m * nv) * 4;
  float x[4] = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < a.ksplit; ++s) {
    const float4 v = *reinterpret_cast<const float4*>(a.partial + ((long)s * a.M + m) * a.N + n);
    x[0] += v.x; x[1] += v.y; x[2] += v.z; x[3] += v.w;
  }
  epilogue4<bf16>(a.epi, m, n, x);
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

static bool fast_seg(const ASeg& g, int Ho, int Wo, int BK) {
  return g.stride == 1 && !g.up && (g.ks == 1 || g.ks == 2 || g.ks == 3) && g.Hi == Ho && g.Wi == Wo &&
         g.cin % BK == 0 && (g.c1 == 0 || g.c0 % BK == 0) && g.scale == nullptr;
}

// Loader mode of a GEMM (see the kernel); modes 1 and 2 address each source
// with 32-bit byte offsets, so its bytes must stay below 2^31.
static int loader_mode(const GemmArgs& a, int BK) {
  const ASeg& g0 = a.seg[0];
  const long hwo = (long)g0.Ho * g0.Wo;
  if (hwo <= 0 || g0.scale) return 0;
  auto small = [&](const ASeg& g, long npix) {
    return npix * (long)g.c0 * 2 < (1L << 31) && npix * (long)g.c1 * 2 < (1L << 31);
  };
  if (fast_seg(g0, g0.Ho, g0.Wo, BK) && (a.seg[1].K == 0 || fast_seg(a.seg[1], g0.Ho, g0.Wo, BK)) && small(g0, a.M) &&
      (a.seg[1].K == 0 || small(a.seg[1], a.M)) && (long)a.N * a.ldb * 2 < (1L << 31))
    return 1;
  if (a.seg[1].K == 0 && g0.ks == 3 && (g0.stride == 2 || g0.up) && g0.c1 == 0 && g0.cin % BK == 0 &&
      (a.M / hwo) * (long)g0.Hi * g0.Wi * g0.c0 * 2 < (1L << 31) && (long)a.N * a.ldb * 2 < (1L << 31) &&
      g0.Ho < 65536 && g0.Wo < 65536)
    return 2;
  return 0;
}

template <int BM, int BN, int BK, int WM, int WN, int MINB = 1>
static void launch_bf16(const GemmArgs& a, hipStream_t s) {
  const long blocks = (long)((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  const dim3 g((unsigned)blocks), b(256);
  switch (loader_mode(a, BK)) {
    case 1: gemm_bf16_kernel<BM, BN, BK, WM, WN, 1, MINB><<<g, b, 0, s>>>(a); break;
    case 2: gemm_bf16_kernel<BM, BN, BK, WM, WN, 2, MINB><<<g, b, 0, s>>>(a); break;
    default: gemm_bf16_kernel<BM, BN, BK, WM, WN, 0, MINB><<<g, b, 0, s>>>(a); break;
  }
}

// Direct-to-LDS kernel for the uniform-tap modes; false if the layer needs
// the register-staged loader.
template <int BM, int BN, int WM, int WN, int DNS, int MINB, int DK = DKS, bool UNIFORM_ONLY = false>
static bool launch_dma(const GemmArgs& a, hipStream_t s) {
  const int mode = loader_mode(a, DK);
  if (mode == 0 || (UNIFORM_ONLY && mode != 1) || (DK != DKS && a.ksplit > 1)) return false;
  const long blocks = (long)((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN) * a.ksplit;
  const dim3 g((unsigned)blocks), b(64 * WM * WN);
  // K order (see the kernel): channel block outer, taps inner on images
  // larger than 8x8.
  const bool ti = (long)a.seg[0].Ho * a.seg[0].Wo > 64;
  if (mode == 1 && ti)
    gemm_bf16_dma_kernel<BM, BN, WM, WN, 1, DNS, MINB, DK, true><<<g, b, 0, s>>>(a);
  else if (mode == 1)
    gemm_bf16_dma_kernel<BM, BN, WM, WN, 1, DNS, MINB, DK, false><<<g, b, 0, s>>>(a);
  else if constexpr (!UNIFORM_ONLY) {
    if (ti)
      gemm_bf16_dma_kernel<BM, BN, WM, WN, 2, DNS, MINB, DK, true><<<g, b, 0, s>>>(a);
    else
      gemm_bf16_dma_kernel<BM, BN, WM, WN, 2, DNS, MINB, DK, false><<<g, b, 0, s>>>(a);
  }
  if (a.ksplit > 1) {
    const long n = (long)a.M * (a.N / 4);
    splitk_reduce_kernel<<<dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s>>>(a);
  }
  return true;
}

// Split-K factor of a bf16 GEMM: long-K 3x3 convolutions on the small
// levels (16x16 and 8x8 images) have too few output tiles to fill 256 CUs.
// The factor depends only on K and the per-image output size, never on the
// number of rows, so a row's result does not depend on its batch-mates.
// Linear layers (1x1, the row count as image width) are never split: their
// "image" size is the row count.
int gemm_ksplit(const GemmArgs& a) {
  const long hw = (long)a.seg[0].Ho * a.seg[0].Wo;
  if (a.seg[0].ks != 3 || a.K < 5120 || hw > 256 || a.N % 160 || a.epi.geglu || a.epi.vt_out || a.epi.out_f32)
    return 1;
  if (loader_mode(a, DKS) == 0) return 1;
  return hw <= 64 ? 4 : 2;
}

// Tile choice: the widest N tile that divides N (320 and 160 cover every
// SD-1.5 / SDXL width: 320, 640, 1280 and their 2x, 3x, 4x, 8x), then the
// tallest M tile that still gives every CU about two blocks.  The tile shape
// never changes a row's K order, so only the split factor (a function of the
// layer shape) decides a row's bits.
hipError_t launch_gemm(DType dt, const GemmArgs& args, hipStream_t s) {
  GemmArgs a = args;
  if (a.ksplit < 1) a.ksplit = 1;
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (a.ksplit > 1 && (dt != BF16 || !a.partial || a.epi.geglu || a.epi.vt_out || a.epi.out_f32 ||
                       a.N % 160 || loader_mode(a, DKS) == 0))
    return hipErrorInvalidValue;
  if (dt == BF16 && (a.N % 4 || a.epi.ldo % 4 || (a.epi.resid && a.epi.ldr % 4) || (a.epi.geglu && a.N % 32) ||
                     a.epi.qcols % 4))
    return hipErrorInvalidValue;
  if (dt != BF16 && (a.epi.geglu || a.epi.vt_out)) return hipErrorInvalidValue;
  if (a.epi.vt_out && (a.epi.vt_col0 % 8 || a.epi.resid || a.epi.tbias || a.epi.out_f32))
    return hipErrorInvalidValue;
  if (a.epi.rowscale && dt != BF16) return hipErrorInvalidValue;
  if ((long)a.N * a.ldb * (dt == BF16 ? 2 : 4) >= (1L << 31)) return hipErrorInvalidValue;
  // upsample phases (ks 2): bf16, the direct-to-LDS tiles (N % 160) with
  // the uniform-tap loader only
  const bool phased = a.seg[0].ks == 2 || (a.seg[1].K && a.seg[1].ks == 2);
  if (phased && (dt != BF16 || a.N % 160 || loader_mode(a, DKS) != 1 || a.ksplit > 1 || a.seg[1].K))
    return hipErrorInvalidValue;
  if (a.epi.phase && (a.epi.phase > 4 || a.epi.ph_h < 1 || a.epi.ph_w < 1 || a.M % (a.epi.ph_h * a.epi.ph_w) ||
                      a.epi.resid || a.epi.vt_out || a.epi.tbias || a.epi.geglu))
    return hipErrorInvalidValue;
  if (dt == BF16) {
    auto nblk = [&](int bm, int bn) { return (long)((a.M + bm - 1) / bm) * ((a.N + bn - 1) / bn); };
    const long want = 2 * 256;
    // Long-K layers of widths that are multiples of 256 (the 1280-wide
    // levels) may take 256x256 tiles: four waves of 128x128 with the
    // accumulators in AGPRs, one block per CU (3 x 32 KB stages), about 14 %
    // faster per tile-product than two 256x160 blocks per CU.  With one
    // block per CU the last wave of blocks can leave much of the chip idle,
    // so they are taken only where their share of busy block slots, with
    // that margin, is at least the narrower tiles' (two per CU).  Every
    // tile gives the same bits, so the choice may follow the row count.
    auto busy = [](long blocks, long slots) { return (double)blocks / (double)(((blocks + slots - 1) / slots) * slots); };
    const long n_wide = nblk(256, 256) * a.ksplit;
    const long n_alt = (a.N % 160 == 0 ? nblk(256, 160) : nblk(256, 128)) * a.ksplit;
    if (a.N % 256 == 0 && a.K >= 2560 && n_wide >= 128 && 1.1 * busy(n_wide, 256) >= busy(n_alt, 512) &&
        !a.epi.vt_out && !a.epi.out_f32 && !a.epi.geglu && !a.epi.rowscale && a.epi.qcols == 0 &&
        launch_dma<256, 256, 2, 2, 3, 1, DKS, true>(a, s)) {
    } else if (a.N % 160 == 0) {
      // 256x160 tiles through the direct-to-LDS pipeline whenever the loader
      // is uniform: taller tiles cut the weight re-reads that dominate
      // small-M layers.  Three K stages (two for the split-K layers) still
      // leave LDS for two blocks per CU.  Otherwise register-staged 64-deep
      // tiles, one block per CU.
      const bool big = nblk(256, 160) * a.ksplit >= want;
      if (a.ksplit == 1 && nblk(256, 160) < 256 && launch_dma<64, 160, 2, 1, 2, 4>(a, s)) {
        // short M (the context K/V projections): 64-row tiles, four blocks per CU
      } else if (a.ksplit == 1 && launch_dma<256, 160, 4, 1, 3, 2>(a, s)) {
        // three K stages (2 x 79.9 KB of LDS: still two blocks per CU)
      } else if (launch_dma<256, 160, 4, 1, 2, 2>(a, s)) {
      } else if (big) {
        launch_bf16<256, 160, 64, 4, 1>(a, s);
      } else {
        launch_bf16<128, 160, 64, 4, 1>(a, s);
      }
    } else if (a.N % 128 == 0 && a.ksplit == 1 && launch_dma<256, 128, 4, 1, 3, 2>(a, s)) {
      // widths that are multiples of 128 but not of 160 (the VAE decoder's
      // 128 / 256 / 512): the same direct-to-LDS pipeline in 256x128 tiles,
      // waves of 64x128, three K stages (2 x 73.7 KB of LDS)
    } else if (a.N % 128 == 0 || a.N > 64) {
      if (nblk(256, 128) >= want)
        launch_bf16<256, 128, 64, 2, 2>(a, s);
      else if (nblk(128, 128) >= want)
        launch_bf16<128, 128, 64, 2, 2>(a, s);
      else
        launch_bf16<64, 128, 64, 2, 2>(a, s);
    } else if (a.N > 32) {
      launch_bf16<128, 64, 64, 4, 1>(a, s);
    } else {
      launch_bf16<256, 32, 64, 4, 1>(a, s);
    }
  } else {
    const long blocks = (long)((a.M + sf::BM - 1) / sf::BM) * ((a.N + sf::BN - 1) / sf::BN);
    gemm_f32_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(a);
  }
  return hipGetLastError();
}

}  // namespace sd
