// The step's last stage in one kernel (bf16 path): the UNet's output
// convolution (3x3, zero padding 1, C -> 4 channels) for a request's
// conditional and, under CFG, unconditional row, the classifier-free
// guidance combine eps = eps_u + w (eps_c - eps_u) (eps = eps_c under
// Skip-CFG, whose unconditional branch is bypassed: Sec. II-B, Sec. III-B)
// and the DDIM update x' = A x + B eps (eta = 0), all in registers.  The
// per-row eps never reaches memory.
//
// The convolution is computed per input pixel rather than per output pixel:
// for every pixel p of the block's tile (plus one image row and one pixel of
// halo on either side) the MFMAs form the 36 partial products
//     Y[p][tap][o] = sum_c x[p][c] w[o][tap][c]      (tap = 3 ky + kx)
// with the pixel's channels read once, 160 contiguous bytes per lane.  The
// output pixel then sums its 9 taps from LDS,
//     eps[p][o] = b[o] + sum over in-image taps of Y[p + (ky-1) W + (kx-1)][tap][o],
// so the zero padding is the taps that are skipped, and the K reduction over
// channels happens across the lanes of each MFMA.
//
// MFMA v_mfma_f32_16x16x32_bf16 with the weights as the first operand (16
// of the 36 (tap, o) columns per tile, 3 tiles, zero rows past 36) and 16
// pixels as the second; the K slice of lane group g = lane / 16 is channels
// [g C/4, (g+1) C/4), 8 per step, for both operands.  The weights of a
// lane stay in registers for the whole block.
#include "device_common.h"
#include "kernels.h"

namespace sd {

constexpr int OUT_P = 256;  // output pixels per block (one per thread)

template <int S>  // S = C / 32 MFMA steps over the channels
__global__ __launch_bounds__(256, 2) void out_cfg_ddim_kernel(OutArgs a) {
  extern __shared__ __attribute__((aligned(16))) float Y[];  // [pixel - q0][9 taps][4]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, pl = lane & 15;
  const int W = a.W, HW = a.H * a.W, C = a.C, cq = C / 4;
  const int ri = blockIdx.x / a.tiles, tile = blockIdx.x - ri * a.tiles;
  const int r = a.order ? a.order[ri] : ri;
  const int ru = a.req_row_u[r];
  const int p0 = tile * OUT_P, p1 = min(HW, p0 + OUT_P);
  const int q0 = max(0, p0 - W - 1), q1 = min(HW, p1 + W + 1);

  // weight fragments: tile t, row pl is column j = 16 t + pl = (tap j / 4, output j % 4)
  bf16x8 wf[3][S];
#pragma unroll
  for (int t = 0; t < 3; ++t) {
    const int j = 16 * t + pl, tap = j >> 2, o = j & 3;
#pragma unroll
    for (int s = 0; s < S; ++s) {
      bf16x8 v = {};
      if (j < 36) v = *reinterpret_cast<const bf16x8*>(a.w + (long)o * 9 * C + tap * C + g * cq + 8 * s);
      wf[t][s] = v;
    }
  }

  // Y over pixels [q0, q1) of one row: 16-pixel tiles dealt round-robin to
  // the waves, the next tile's loads issued before the current one's MFMAs.
  auto compute_y = [&](int row) {
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(a.x + (long)row * HW * C, (long)HW * C * 2);
    const int ntile = (q1 - q0 + 15) >> 4;
    bf16x8 cur[S], nxt[S];
    auto fetch = [&](int tt, bf16x8(&v)[S]) {
      const int px = q0 + 16 * tt + pl;
      const bool ok = px < q1;
      const int off = (px * C + g * cq) * 2;
#pragma unroll
      for (int s = 0; s < S; ++s) v[s] = buf_load16(rs, ok ? off + 16 * s : OOB);
    };
    if (wave < ntile) fetch(wave, cur);
    for (int tt = wave; tt < ntile; tt += 4) {
      if (tt + 4 < ntile) fetch(tt + 4, nxt);
      f32x4 acc[3];
#pragma unroll
      for (int t = 0; t < 3; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < S; ++s)
#pragma unroll
        for (int t = 0; t < 3; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[t][s], cur[s], acc[t], 0, 0, 0);
      // lane (g, pl) holds rows 4 g .. 4 g + 3 of each tile = tap 4 t + g, outputs 0..3, of pixel pl
      const int px = q0 + 16 * tt + pl;
      if (px < q1) {
#pragma unroll
        for (int t = 0; t < 3; ++t)
          if (4 * t + g < 9)
            *reinterpret_cast<f32x4*>(&Y[(px - q0) * 36 + (4 * t + g) * 4]) = acc[t];
      }
#pragma unroll
      for (int s = 0; s < S; ++s) cur[s] = nxt[s];
    }
  };
  // eps of this thread's output pixel: bias plus its in-image taps
  const int p = p0 + tid;
  auto gather = [&](float e[4]) {
#pragma unroll
    for (int o = 0; o < 4; ++o) e[o] = a.bias[o];
    if (p >= p1) return;
    const int y = p / W, x = p - y * W;
#pragma unroll
    for (int ky = 0; ky < 3; ++ky) {
      const int yy = y + ky - 1;
      if (yy < 0 || yy >= a.H) continue;
#pragma unroll
      for (int kx = 0; kx < 3; ++kx) {
        const int xx = x + kx - 1;
        if (xx < 0 || xx >= W) continue;
        const f32x4 v = *reinterpret_cast<const f32x4*>(&Y[(p + (ky - 1) * W + (kx - 1) - q0) * 36 + (3 * ky + kx) * 4]);
#pragma unroll
        for (int o = 0; o < 4; ++o) e[o] += v[o];
      }
    }
  };

  float ec[4], eu[4];
  compute_y(r);
  __syncthreads();
  gather(ec);
  if (ru >= 0) {
    __syncthreads();  // every thread has read the conditional row's Y
    compute_y(ru);
    __syncthreads();
    gather(eu);
  }
  if (p < p1) {
    const float A = a.req_coef[3 * r], B = a.req_coef[3 * r + 1], w = a.req_coef[3 * r + 2];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      float e = ec[c];
      if (ru >= 0) e = eu[c] + w * (e - eu[c]);
      const long o = ((long)r * 4 + c) * HW + p;
      a.lat_out[o] = A * a.lat_in[o] + B * e;
      if (a.eps_out) a.eps_out[o] = e;
    }
  }
}

bool out_cfg_ddim_ok(DType dt, int latent_c, int H, int W, int C) {
  return dt == BF16 && latent_c == 4 && H >= 1 && W >= 1 && W <= 128 && C >= 32 && C <= 320 && C % 32 == 0 &&
         (long)H * W * C * 2 < (1L << 31);
}

size_t out_cfg_ddim_lds_bytes(int W) { return (size_t)(OUT_P + 2 * W + 2) * 36 * sizeof(float); }

template <int S>
static hipError_t launch_out_s(const OutArgs& a, unsigned blocks, size_t lds, hipStream_t s) {
  if (lds > 64 * 1024) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&out_cfg_ddim_kernel<S>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  out_cfg_ddim_kernel<S><<<blocks, 256, lds, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_out_cfg_ddim(const OutArgs& args, hipStream_t s) {
  OutArgs a = args;
  if (!out_cfg_ddim_ok(BF16, 4, a.H, a.W, a.C) || a.n_req < 0) return hipErrorInvalidValue;
  const int HW = a.H * a.W;
  a.tiles = (HW + OUT_P - 1) / OUT_P;
  if (a.n_req == 0) return hipSuccess;
  const long blocks = (long)a.n_req * a.tiles;
  if (blocks > 0x7FFFFFFFL) return hipErrorInvalidValue;
  const size_t lds = out_cfg_ddim_lds_bytes(a.W);
  switch (a.C / 32) {
    case 1: return launch_out_s<1>(a, (unsigned)blocks, lds, s);
    case 2: return launch_out_s<2>(a, (unsigned)blocks, lds, s);
    case 3: return launch_out_s<3>(a, (unsigned)blocks, lds, s);
    case 4: return launch_out_s<4>(a, (unsigned)blocks, lds, s);
    case 5: return launch_out_s<5>(a, (unsigned)blocks, lds, s);
    case 6: return launch_out_s<6>(a, (unsigned)blocks, lds, s);
    case 7: return launch_out_s<7>(a, (unsigned)blocks, lds, s);
    case 8: return launch_out_s<8>(a, (unsigned)blocks, lds, s);
    case 9: return launch_out_s<9>(a, (unsigned)blocks, lds, s);
    case 10: return launch_out_s<10>(a, (unsigned)blocks, lds, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace sd
