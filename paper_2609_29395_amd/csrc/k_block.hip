// Data movement of the ResNet basic block (the paper's ResNet-18, Sec. V-A):
// the strided convolutions run as dense products on the conv kernels' own
// MFMA tiles, and these kernels stage their operands.
//
//   im2col       a strided conv's input as rows of its R x S taps: row
//                (b, ho, wo), column (r, s, c) = x[b][ho*stride + r - pad]
//                [wo*stride + s - pad][c], zero outside the image and in the
//                padding columns up to Kc.  The forward and the weight
//                gradient then take these rows as a one-tap product.
//   zero_insert  a stride-2 conv's output gradient spread back to the input
//                grid: gup[b][h][w] = g[b][h/2][w/2] at even (h, w), zero
//                elsewhere.  The input gradient of a 3x3 / pad 1 (or 1x1 /
//                pad 0) conv with stride 2 is then the stride-1 input
//                gradient of gup (the inserted zeros add exact zeros), on
//                the stride-1 kernels.
// One 16-byte vector of channels per thread; grid (vectors / 256, replica
// slots).  Channel counts are multiples of the vector width.
#include "runtime.h"

namespace {

template <typename T>
__global__ void __launch_bounds__(256)
im2col_kernel(const T *__restrict__ x, T *__restrict__ cols, const int32_t *__restrict__ rmap, int64_t x_rs,
              int64_t c_rs, uint32_t total, int H, int W, int Ci, int Ho, int Wo, int R, int S, int stride, int pad,
              int Kc) {
  constexpr int VEC = ElemT<T>::VEC;
  const uint32_t i = blockIdx.x * 256u + threadIdx.x;
  if (i >= total) return;
  const int rep = replica_of(rmap, blockIdx.y);
  const int KV = Kc / VEC;
  const uint32_t row = i / (uint32_t)KV;
  const int k = (int)(i - row * (uint32_t)KV) * VEC;
  const int wo = (int)(row % (uint32_t)Wo);
  const uint32_t q = row / (uint32_t)Wo;
  const int ho = (int)(q % (uint32_t)Ho), b = (int)(q / (uint32_t)Ho);
  uint4 v = make_uint4(0u, 0u, 0u, 0u);
  if (k < R * S * Ci) {
    const int rs = k / Ci, c = k - rs * Ci;
    const int r = rs / S, s = rs - r * S;
    const int h = ho * stride + r - pad, w = wo * stride + s - pad;
    if ((unsigned)h < (unsigned)H && (unsigned)w < (unsigned)W)
      v = *reinterpret_cast<const uint4 *>(x + rep * x_rs + (((int64_t)b * H + h) * W + w) * Ci + c);
  }
  *reinterpret_cast<uint4 *>(cols + rep * c_rs + (int64_t)row * Kc + k) = v;
}

template <typename T>
__global__ void __launch_bounds__(256)
zero_insert_kernel(const T *__restrict__ g, T *__restrict__ gup, const int32_t *__restrict__ rmap, int64_t g_rs,
                   int64_t u_rs, uint32_t total, int H, int W, int Ho, int Wo, int Ch) {
  constexpr int VEC = ElemT<T>::VEC;
  const uint32_t i = blockIdx.x * 256u + threadIdx.x;
  if (i >= total) return;
  const int rep = replica_of(rmap, blockIdx.y);
  const int CV = Ch / VEC;
  const uint32_t px = i / (uint32_t)CV;
  const int c = (int)(i - px * (uint32_t)CV) * VEC;
  const int w = (int)(px % (uint32_t)W);
  const uint32_t q = px / (uint32_t)W;
  const int h = (int)(q % (uint32_t)H), b = (int)(q / (uint32_t)H);
  uint4 v = make_uint4(0u, 0u, 0u, 0u);
  if (!(h & 1) && !(w & 1) && (h >> 1) < Ho && (w >> 1) < Wo)
    v = *reinterpret_cast<const uint4 *>(g + rep * g_rs + (((int64_t)b * Ho + (h >> 1)) * Wo + (w >> 1)) * Ch + c);
  *reinterpret_cast<uint4 *>(gup + rep * u_rs + (int64_t)px * Ch + c) = v;
}

}  // namespace

hipError_t launch_im2col(int dtype, const void *x, void *cols, int C, const int32_t *rmap, int Bt, int H, int W,
                         int Ci, int Ho, int Wo, int R, int S, int stride, int pad, int Kc, hipStream_t s) {
  const int vec = dtype == GCPSL_BF16 ? 8 : 4;
  if (Ci % vec || Kc % vec || Kc < R * S * Ci) return hipErrorInvalidValue;
  const uint32_t total = (uint32_t)((int64_t)Bt * Ho * Wo * (Kc / vec));
  const dim3 g((total + 255) / 256, C);
  const int64_t x_rs = (int64_t)Bt * H * W * Ci, c_rs = (int64_t)Bt * Ho * Wo * Kc;
  if (dtype == GCPSL_BF16)
    hipLaunchKernelGGL(im2col_kernel<bf16_t>, g, dim3(256), 0, s, (const bf16_t *)x, (bf16_t *)cols, rmap, x_rs, c_rs,
                       total, H, W, Ci, Ho, Wo, R, S, stride, pad, Kc);
  else
    hipLaunchKernelGGL(im2col_kernel<float>, g, dim3(256), 0, s, (const float *)x, (float *)cols, rmap, x_rs, c_rs,
                       total, H, W, Ci, Ho, Wo, R, S, stride, pad, Kc);
  return hipGetLastError();
}

hipError_t launch_zero_insert(int dtype, const void *g, void *gup, int C, const int32_t *rmap, int Bt, int H, int W,
                              int Ho, int Wo, int Ch, hipStream_t s) {
  const int vec = dtype == GCPSL_BF16 ? 8 : 4;
  if (Ch % vec) return hipErrorInvalidValue;
  const uint32_t total = (uint32_t)((int64_t)Bt * H * W * (Ch / vec));
  const dim3 grid((total + 255) / 256, C);
  const int64_t g_rs = (int64_t)Bt * Ho * Wo * Ch, u_rs = (int64_t)Bt * H * W * Ch;
  if (dtype == GCPSL_BF16)
    hipLaunchKernelGGL(zero_insert_kernel<bf16_t>, grid, dim3(256), 0, s, (const bf16_t *)g, (bf16_t *)gup, rmap,
                       g_rs, u_rs, total, H, W, Ho, Wo, Ch);
  else
    hipLaunchKernelGGL(zero_insert_kernel<float>, grid, dim3(256), 0, s, (const float *)g, (float *)gup, rmap, g_rs,
                       u_rs, total, H, W, Ho, Wo, Ch);
  return hipGetLastError();
}
