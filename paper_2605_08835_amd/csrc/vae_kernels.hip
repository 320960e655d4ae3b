// Kernels of the VAE decoder that the UNet step has no counterpart for: the
// decoder's input (latent scaling + the 1x1 post-quantisation conv, packed
// channels-last), the row softmax of its single-head mid-block attention,
// and the image write-out.  The decoder's convolutions, GroupNorms and
// linears run on the UNet step's kernels.
#include "device_common.h"
#include "kernels.h"

namespace sd {

// y[i, p, o] = b[o] + sum_c w[o, c] (lat[i, c, p] * inv_scale) for o < lc,
// 0 for lc <= o < cpad (channels-last, padded for 16-byte loads).
template <typename T>
__global__ void vae_input_kernel(const float* lat, const float* w, const float* b, float inv_scale, T* y,
                                 int n, int lc, int hw, int cpad) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long)n * hw) return;
  const int img = (int)(i / hw), p = (int)(i - (long)img * hw);
  float z[8];
  for (int c = 0; c < lc; ++c) z[c] = lat[((long)img * lc + c) * hw + p] * inv_scale;
  for (int o = 0; o < cpad; ++o) {
    float v = 0.f;
    if (o < lc) {
      v = b[o];
      for (int c = 0; c < lc; ++c) v = fmaf(w[o * lc + c], z[c], v);
    }
    y[i * cpad + o] = from_f<T>(v);
  }
}

hipError_t launch_vae_input(DType dt, const float* lat, const float* w, const float* b, float inv_scale, void* y,
                            int n, int lc, int hw, int cpad, hipStream_t s) {
  const long total = (long)n * hw;
  if (total == 0) return hipSuccess;
  if (lc > 8 || cpad < lc) return hipErrorInvalidValue;
  const unsigned blocks = (unsigned)((total + 255) / 256);
  if (dt == BF16)
    vae_input_kernel<bf16><<<blocks, 256, 0, s>>>(lat, w, b, inv_scale, (bf16*)y, n, lc, hw, cpad);
  else
    vae_input_kernel<float><<<blocks, 256, 0, s>>>(lat, w, b, inv_scale, (float*)y, n, lc, hw, cpad);
  return hipGetLastError();
}

// P[r, :] = softmax(scale * S[r, :]) for fp32 scores S [rows, cols]; one
// block of 256 threads per row, the row in registers (cols <= 256 * 32),
// max and sum reduced in fp32 across the block.
template <typename T, int PER>
__global__ __launch_bounds__(256) void softmax_rows_kernel(const float* S, T* P, int cols, float scale) {
  __shared__ float red[2][4];
  const long row = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* s = S + row * cols;
  float v[PER];
  float m = -3.0e38f;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int c = tid + 256 * e;
    v[e] = c < cols ? s[c] * scale : -3.0e38f;
    m = fmaxf(m, v[e]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
  if (lane == 0) red[0][wave] = m;
  __syncthreads();
  m = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));
  float sum = 0.f;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int c = tid + 256 * e;
    v[e] = c < cols ? __expf(v[e] - m) : 0.f;
    sum += v[e];
  }
  sum = wave_sum(sum);
  if (lane == 0) red[1][wave] = sum;
  __syncthreads();
  const float inv = 1.0f / (red[1][0] + red[1][1] + red[1][2] + red[1][3]);
  T* p = P + row * cols;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int c = tid + 256 * e;
    if (c < cols) p[c] = from_f<T>(v[e] * inv);
  }
}

hipError_t launch_softmax_rows(DType dt, const float* S, void* P, long rows, int cols, float scale, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (cols < 1 || cols > 256 * 32 || rows > 0x7FFFFFFFL) return hipErrorInvalidValue;
  const unsigned g = (unsigned)rows;
  const int per = (cols + 255) / 256;
#define SD_SOFTMAX(PER)                                                                          \
  if (dt == BF16)                                                                                \
    softmax_rows_kernel<bf16, PER><<<g, 256, 0, s>>>(S, (bf16*)P, cols, scale);                  \
  else                                                                                           \
    softmax_rows_kernel<float, PER><<<g, 256, 0, s>>>(S, (float*)P, cols, scale);
  if (per <= 1) {
    SD_SOFTMAX(1)
  } else if (per <= 4) {
    SD_SOFTMAX(4)
  } else if (per <= 16) {
    SD_SOFTMAX(16)
  } else {
    SD_SOFTMAX(32)
  }
#undef SD_SOFTMAX
  return hipGetLastError();
}

// img[i, c, p] = y[i, p, c] for c < oc (channels-last fp32 with ld channels
// per pixel -> NCHW fp32).
__global__ void image_out_kernel(const float* y, float* img, int n, int hw, int ld, int oc) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long)n * hw) return;
  const int im = (int)(i / hw), p = (int)(i - (long)im * hw);
  for (int c = 0; c < oc; ++c) img[((long)im * oc + c) * hw + p] = y[i * ld + c];
}

hipError_t launch_image_out(const float* y, float* img, int n, int hw, int ld, int oc, hipStream_t s) {
  const long total = (long)n * hw;
  if (total == 0) return hipSuccess;
  image_out_kernel<<<(unsigned)((total + 255) / 256), 256, 0, s>>>(y, img, n, hw, ld, oc);
  return hipGetLastError();
}

}  // namespace sd
