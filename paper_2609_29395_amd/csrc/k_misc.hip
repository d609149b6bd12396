// Sampling, gather, pools, the classifier head, SGD and fusion kernels.
#include "rng.h"
#include "runtime.h"

namespace {

constexpr int kMaxBitmapWords = 2048;  // clients tracked per cluster: K <= 65536

// ---------------------------------------------------------------- sampling
// Eq. 1 / Eq. 3: cluster n's batch at local round `step` is B distinct
// examples of its own pool: positions [tB, (t+1)B) of the keyed permutation
// of epoch e = step / S_n, S_n = floor(n_n / B).  Also counts the distinct
// clients of the batch, |A_{n,t}| (Sec. III-A).
__global__ void __launch_bounds__(256)
sample_kernel(const int32_t *__restrict__ ids, const int64_t *__restrict__ off,
              const int32_t *__restrict__ coe, const int32_t *__restrict__ labels,
              int32_t *__restrict__ idx, int32_t *__restrict__ y, int32_t *__restrict__ hits,
              int C, int B, int K, uint64_t seed, int64_t step0, int64_t max_steps) {
  __shared__ uint32_t bitmap[kMaxBitmapWords];
  __shared__ int count;
  const int n = blockIdx.x, j = blockIdx.y, tid = threadIdx.x;
  const int64_t step = step0 + j;
  const int64_t lo = off[n];
  const uint32_t nn = (uint32_t)(off[n + 1] - lo);
  const int64_t S = nn / (uint32_t)B;
  const int64_t e = step / S, t = step % S;
  const uint64_t key = gc_sample_key(seed, (uint64_t)n, (uint64_t)e);
  const int words = (K + 31) >> 5;
  for (int w = tid; w < words; w += blockDim.x) bitmap[w] = 0u;
  if (tid == 0) count = 0;
  __syncthreads();
  for (int i = tid; i < B; i += blockDim.x) {
    const uint32_t p = (uint32_t)(t * B + i);
    const int32_t ex = ids[lo + gc_permute(p, nn, key)];
    const int64_t o = ((int64_t)j * C + n) * B + i;
    idx[o] = ex;
    y[o] = labels[ex];
    const int32_t c = coe[ex];
    atomicOr(&bitmap[c >> 5], 1u << (c & 31));
  }
  __syncthreads();
  int local = 0;
  for (int w = tid; w < words; w += blockDim.x) local += __popc(bitmap[w]);
  atomicAdd(&count, local);
  __syncthreads();
  if (tid == 0 && step < max_steps) hits[step * C + n] = count;
}

template <typename T>
__global__ void __launch_bounds__(256)
gather_kernel(const float *__restrict__ images, const int32_t *__restrict__ idx, T *__restrict__ x,
              int64_t row_elems) {
  const int64_t row = blockIdx.x;
  const float *src = images + (int64_t)idx[row] * row_elems;
  T *dst = x + row * row_elems;
  if ((row_elems & 3) == 0) {
    const int64_t nv = row_elems >> 2;
    for (int64_t v = threadIdx.x; v < nv; v += blockDim.x) {
      const float4 f = reinterpret_cast<const float4 *>(src)[v];
      if constexpr (sizeof(T) == 4) {
        reinterpret_cast<float4 *>(dst)[v] = f;
      } else {
        const uint32_t lo = (uint32_t)f32_to_bf16(f.x) | ((uint32_t)f32_to_bf16(f.y) << 16);
        const uint32_t hi = (uint32_t)f32_to_bf16(f.z) | ((uint32_t)f32_to_bf16(f.w) << 16);
        reinterpret_cast<uint2 *>(dst)[v] = make_uint2(lo, hi);
      }
    }
  } else {
    for (int64_t v = threadIdx.x; v < row_elems; v += blockDim.x) dst[v] = ElemT<T>::from_f(src[v]);
  }
}

// Gather for a first layer with few channels: each staged pixel holds its
// 3x3 neighbourhood (k = (r, s, c), zero outside the image and beyond 9 Cin
// up to Kc), so that layer runs as a plain GEMM with K = Kc.  The image is
// staged in LDS when it fits.
template <typename T>
__global__ void __launch_bounds__(256)
gather_im2col_kernel(const float *__restrict__ images, const int32_t *__restrict__ idx,
                     T *__restrict__ x, int H, int W, int Cin, int Kc, int use_lds) {
  extern __shared__ float img[];
  constexpr int VEC = ElemT<T>::VEC;
  const int64_t row = blockIdx.x;
  const int64_t n = (int64_t)H * W * Cin;
  const float *src = images + (int64_t)idx[row] * n;
  if (use_lds) {
    for (int64_t i = threadIdx.x; i < n; i += blockDim.x) img[i] = src[i];
    __syncthreads();
  }
  const float *from = use_lds ? img : src;
  T *dst = x + row * (int64_t)H * W * Kc;
  const int K9 = 9 * Cin;
  for (int p = threadIdx.x; p < H * W; p += blockDim.x) {
    const int h = p / W, w = p % W;
    for (int k0 = 0; k0 < Kc; k0 += VEC) {
      struct { T v[VEC]; } pk;
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const int k = k0 + e;
        float v = 0.f;
        if (k < K9) {
          const int rs = k / Cin, c = k - rs * Cin;
          const int hh = h + rs / 3 - 1, ww = w + rs % 3 - 1;
          if ((unsigned)hh < (unsigned)H && (unsigned)ww < (unsigned)W) v = from[(hh * W + ww) * Cin + c];
        }
        pk.v[e] = ElemT<T>::from_f(v);
      }
      *reinterpret_cast<uint4 *>(dst + (int64_t)p * Kc + k0) = __builtin_bit_cast(uint4, pk);
    }
  }
}

// ------------------------------------------------------ weight preparation
// Compute copies of one conv layer's weights from the fp32 masters:
//   wf[co][k], k = (r, s, ci) < 9 ci, rows zero-padded to Kp (forward);
//   wd[ci][kk], kk = (r', s', co), wd[ci][(r', s', co)] = W[co][2-r'][2-s'][ci]
//   rows zero-padded to Kdp (input gradient as a forward conv).
// wf is a row copy; wd is a transpose of 64 x 64 (co, ci) blocks per kernel
// tap, staged through LDS so both the reads and the writes are coalesced.
template <typename T>
__global__ void __launch_bounds__(256)
prep_wf_kernel(const float *__restrict__ theta, int64_t P, int64_t w_off, int co, int ci,
               T *__restrict__ wf, int Kp) {
  const int rep = blockIdx.y;
  const float *w = theta + rep * P + w_off;
  const int K = 9 * ci;
  const int64_t nf = (int64_t)co * Kp;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < nf;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int n = (int)(i / Kp), k = (int)(i % Kp);
    wf[rep * nf + i] = ElemT<T>::from_f(k < K ? w[(int64_t)n * K + k] : 0.f);
  }
}

template <typename T>
__global__ void __launch_bounds__(256)
prep_wd_kernel(const float *__restrict__ theta, int64_t P, int64_t w_off, int co, int ci,
               T *__restrict__ wd, int Kdp) {
  __shared__ float tile[64][65];
  const int rep = blockIdx.z;
  const int tap = blockIdx.y;  // (r', s') of the flipped kernel
  const int nco = (co + 63) / 64;
  const int cb = blockIdx.x % nco, ib = blockIdx.x / nco;
  const int rs_src = 8 - tap;  // (2 - r') * 3 + (2 - s')
  const float *w = theta + rep * P + w_off;
  const int K = 9 * ci;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int r = ty; r < 64; r += 4) {
    const int o = cb * 64 + r, c = ib * 64 + tx;
    tile[r][tx] = (o < co && c < ci) ? w[(int64_t)o * K + rs_src * ci + c] : 0.f;
  }
  __syncthreads();
  T *dst = wd + (int64_t)rep * ci * Kdp;
  for (int r = ty; r < 64; r += 4) {
    const int c = ib * 64 + r, o = cb * 64 + tx;
    if (c < ci && o < co) dst[(int64_t)c * Kdp + tap * co + o] = ElemT<T>::from_f(tile[tx][r]);
  }
  // zero the row padding once per row (by the first tap/co block)
  if (tap == 0 && cb == 0) {
    for (int r = ty; r < 64; r += 4) {
      const int c = ib * 64 + r;
      if (c >= ci) continue;
      for (int k = 9 * co + tx; k < Kdp; k += 64) dst[(int64_t)c * Kdp + k] = T(0);
    }
  }
}

// -------------------------------------------------------------- max pool
// 2x2 / stride 2 over a [N][H][W][Ch] batch (N = C * B).  The backward pass
// routes each pooled gradient to the first maximum of its window in
// row-major order (strict >) and applies the producing conv's ReLU mask
// (output > 0).
template <typename T>
__global__ void __launch_bounds__(256)
maxpool_fwd_kernel(const T *__restrict__ x, T *__restrict__ z, int64_t total, int H, int W, int Ch) {
  const int Ho = H >> 1, Wo = W >> 1;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(i % Ch);
    int64_t r = i / Ch;
    const int wo = (int)(r % Wo);
    r /= Wo;
    const int ho = (int)(r % Ho);
    const int64_t bi = r / Ho;
    const int64_t base = ((bi * H + 2 * ho) * W + 2 * wo) * Ch + c;
    float m = ElemT<T>::to_f(x[base]);
    T best = x[base];
    const int64_t o[3] = {base + Ch, base + (int64_t)W * Ch, base + (int64_t)W * Ch + Ch};
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      const float v = ElemT<T>::to_f(x[o[q]]);
      if (v > m) {
        m = v;
        best = x[o[q]];
      }
    }
    z[i] = best;
  }
}

template <typename T>
__global__ void __launch_bounds__(256)
maxpool_bwd_kernel(const T *__restrict__ a, const T *__restrict__ gz, T *__restrict__ gpre,
                   int64_t total, int H, int W, int Ch) {
  const int Ho = H >> 1, Wo = W >> 1;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(i % Ch);
    int64_t r = i / Ch;
    const int wo = (int)(r % Wo);
    r /= Wo;
    const int ho = (int)(r % Ho);
    const int64_t bi = r / Ho;
    const int64_t base = ((bi * H + 2 * ho) * W + 2 * wo) * Ch + c;
    const int64_t o[4] = {base, base + Ch, base + (int64_t)W * Ch, base + (int64_t)W * Ch + Ch};
    float v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = ElemT<T>::to_f(a[o[q]]);
    int arg = 0;
#pragma unroll
    for (int q = 1; q < 4; ++q)
      if (v[q] > v[arg]) arg = q;
    const T g = gz[i];
#pragma unroll
    for (int q = 0; q < 4; ++q) gpre[o[q]] = (q == arg && v[q] > 0.f) ? g : T(0);
  }
}

// ------------------------------------------------------------------ head
// Pooled feature h[n][c] = mean over positions of (optionally 2x2-max-pooled)
// last conv output.
template <typename T>
__global__ void __launch_bounds__(256)
head_pool_kernel(const T *__restrict__ a, T *__restrict__ h, int64_t total, int H, int W, int Ch,
                 int maxpool) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(i % Ch);
    const int64_t bi = i / Ch;
    const T *src = a + bi * H * W * Ch + c;
    float s = 0.f;
    int npos;
    if (maxpool) {
      const int Ho = H >> 1, Wo = W >> 1;
      npos = Ho * Wo;
      for (int ho = 0; ho < Ho; ++ho)
        for (int wo = 0; wo < Wo; ++wo) {
          const int64_t b0 = ((int64_t)(2 * ho) * W + 2 * wo) * Ch;
          float m = ElemT<T>::to_f(src[b0]);
          m = fmaxf(m, ElemT<T>::to_f(src[b0 + Ch]));
          m = fmaxf(m, ElemT<T>::to_f(src[b0 + (int64_t)W * Ch]));
          m = fmaxf(m, ElemT<T>::to_f(src[b0 + (int64_t)W * Ch + Ch]));
          s += m;
        }
    } else {
      npos = H * W;
      for (int p = 0; p < npos; ++p) s += ElemT<T>::to_f(src[(int64_t)p * Ch]);
    }
    h[i] = ElemT<T>::from_f(s / (float)npos);
  }
}

// Linear layer and mean softmax cross-entropy for one replica per workgroup:
// logits = h W^T + b, loss = mean_b (logsumexp - logit_y),
// dlogits = (softmax - onehot) / B, dW = dlogits^T h, db = sum_b dlogits,
// dh = dlogits W.  bf16 workloads use the bf16-rounded weight matrix.  The
// pooled features, the weights and the logits are staged in LDS so every
// global access is coalesced; each sum runs in a fixed order.
template <typename T>
__global__ void __launch_bounds__(1024)
linear_ce_kernel(const T *__restrict__ h, const int32_t *__restrict__ y,
                 const float *__restrict__ theta, int64_t P, int64_t w_off, int64_t b_off,
                 float *__restrict__ grad, float *__restrict__ dh, float *__restrict__ loss, int Bt,
                 int Ch, int L) {
  extern __shared__ float sh[];
  float *hs = sh;                      // [Bt][Ch]
  float *ws = hs + (int64_t)Bt * Ch;   // [L][Ch]
  float *lg = ws + (int64_t)L * Ch;    // [Bt][L] logits, then dlogits
  float *lossb = lg + Bt * L;          // [Bt]
  const int rep = blockIdx.x, tid = threadIdx.x, nt = blockDim.x;
  const T *hr = h + (int64_t)rep * Bt * Ch;
  const float *Wl = theta + rep * P + w_off;
  const float *bl = theta + rep * P + b_off;
  for (int i = tid; i < Bt * Ch; i += nt) hs[i] = ElemT<T>::to_f(hr[i]);
  for (int i = tid; i < L * Ch; i += nt) ws[i] = ElemT<T>::to_f(ElemT<T>::from_f(Wl[i]));
  __syncthreads();
  for (int i = tid; i < Bt * L; i += nt) {
    const int b = i / L, j = i % L;
    const float *hb = hs + (int64_t)b * Ch, *wj = ws + (int64_t)j * Ch;
    float s = bl[j];
    for (int c = 0; c < Ch; ++c) s += hb[c] * wj[c];
    lg[i] = s;
  }
  __syncthreads();
  for (int b = tid; b < Bt; b += nt) {
    float m = lg[b * L];
    for (int j = 1; j < L; ++j) m = fmaxf(m, lg[b * L + j]);
    float s = 0.f;
    for (int j = 0; j < L; ++j) s += expf(lg[b * L + j] - m);
    const float lse = logf(s);
    const int yb = y[(int64_t)rep * Bt + b];
    lossb[b] = lse - (lg[b * L + yb] - m);
    for (int j = 0; j < L; ++j) {
      const float p = expf(lg[b * L + j] - m - lse);
      lg[b * L + j] = (p - (j == yb ? 1.f : 0.f)) / (float)Bt;
    }
  }
  __syncthreads();
  if (tid == 0) {
    float s = 0.f;
    for (int b = 0; b < Bt; ++b) s += lossb[b];
    loss[rep] = s / (float)Bt;
  }
  float *g = grad + rep * P;
  for (int i = tid; i < L * Ch; i += nt) {
    const int j = i / Ch, c = i % Ch;
    float s = 0.f;
    for (int b = 0; b < Bt; ++b) s += lg[b * L + j] * hs[(int64_t)b * Ch + c];
    g[w_off + i] = s;
  }
  for (int j = tid; j < L; j += nt) {
    float s = 0.f;
    for (int b = 0; b < Bt; ++b) s += lg[b * L + j];
    g[b_off + j] = s;
  }
  float *dhr = dh + (int64_t)rep * Bt * Ch;
  for (int i = tid; i < Bt * Ch; i += nt) {
    const int b = i / Ch, c = i % Ch;
    float s = 0.f;
    for (int j = 0; j < L; ++j) s += lg[b * L + j] * ws[(int64_t)j * Ch + c];
    dhr[i] = s;
  }
}

// Gradient of the head pooling, with the last conv's ReLU mask:
// gpre = mask * route(dh / npos) (route = first maximum if max pooled).
template <typename T>
__global__ void __launch_bounds__(256)
head_pool_bwd_kernel(const T *__restrict__ a, const float *__restrict__ dh, T *__restrict__ gpre,
                     int64_t total, int H, int W, int Ch, int maxpool) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(i % Ch);
    int64_t r = i / Ch;
    if (maxpool) {
      const int Ho = H >> 1, Wo = W >> 1;
      const int wo = (int)(r % Wo);
      r /= Wo;
      const int ho = (int)(r % Ho);
      const int64_t bi = r / Ho;
      const T g = ElemT<T>::from_f(dh[bi * Ch + c] / (float)(Ho * Wo));
      const int64_t base = ((bi * H + 2 * ho) * W + 2 * wo) * Ch + c;
      const int64_t o[4] = {base, base + Ch, base + (int64_t)W * Ch, base + (int64_t)W * Ch + Ch};
      float v[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) v[q] = ElemT<T>::to_f(a[o[q]]);
      int arg = 0;
#pragma unroll
      for (int q = 1; q < 4; ++q)
        if (v[q] > v[arg]) arg = q;
#pragma unroll
      for (int q = 0; q < 4; ++q) gpre[o[q]] = (q == arg && v[q] > 0.f) ? g : T(0);
    } else {
      const int64_t bi = r / ((int64_t)H * W);
      const T g = ElemT<T>::from_f(dh[bi * Ch + c] / (float)(H * W));
      gpre[i] = ElemT<T>::to_f(a[i]) > 0.f ? g : T(0);
    }
  }
}

// ----------------------------------------------------- split-K reduction
// grad[w_off + j] = sum over splits (in order) of the partial weight
// gradients; grad[b_off + c] likewise for the bias.
__global__ void __launch_bounds__(256)
wgrad_reduce_kernel(const float *__restrict__ dw, const float *__restrict__ db, int splits,
                    int64_t dw_ss, int64_t dw_rs, int64_t db_ss, int64_t db_rs,
                    float *__restrict__ grad, int64_t P, int64_t w_off, int64_t b_off, int64_t nw,
                    int co) {
  const int rep = blockIdx.y;
  for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < nw + co;
       j += (int64_t)gridDim.x * blockDim.x) {
    float s = 0.f;
    if (j < nw) {
      for (int k = 0; k < splits; ++k) s += dw[k * dw_ss + rep * dw_rs + j];
      grad[rep * P + w_off + j] = s;
    } else {
      const int64_t c = j - nw;
      for (int k = 0; k < splits; ++k) s += db[k * db_ss + rep * db_rs + c];
      grad[rep * P + b_off + c] = s;
    }
  }
}

// ------------------------------------------------------------------- SGD
__global__ void __launch_bounds__(256)
sgd_kernel(float *__restrict__ theta, float *__restrict__ mom, const float *__restrict__ grad,
           int64_t n, float lr, float mu) {
  const int64_t nv = n >> 2;
  float4 *t4 = reinterpret_cast<float4 *>(theta);
  float4 *m4 = reinterpret_cast<float4 *>(mom);
  const float4 *g4 = reinterpret_cast<const float4 *>(grad);
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < nv;
       i += (int64_t)gridDim.x * blockDim.x) {
    float4 v = m4[i], t = t4[i];
    const float4 g = g4[i];
    v.x = mu * v.x + g.x; v.y = mu * v.y + g.y; v.z = mu * v.z + g.z; v.w = mu * v.w + g.w;
    t.x -= lr * v.x; t.y -= lr * v.y; t.z -= lr * v.z; t.w -= lr * v.w;
    m4[i] = v;
    t4[i] = t;
  }
  for (int64_t i = 4 * nv + blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const float v = mu * mom[i] + grad[i];
    mom[i] = v;
    theta[i] -= lr * v;
  }
}

// ---------------------------------------------------------------- fusion
// Eq. 5: theta_bar[p] = (sum_n w_n theta_n[p]) / W in fp64, in cluster order,
// rounded once to fp32 and written back to every replica.
__global__ void __launch_bounds__(256)
fuse_kernel(float *__restrict__ theta, const double *__restrict__ w, double W, int C, int64_t P) {
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < P;
       p += (int64_t)gridDim.x * blockDim.x) {
    double acc = 0.0;
    for (int n = 0; n < C; ++n) acc += w[n] * (double)theta[n * P + p];
    const float v = (float)(acc / W);
    for (int n = 0; n < C; ++n) theta[n * P + p] = v;
  }
}

inline unsigned grid_for(int64_t n, int per = 256, unsigned cap = 65535u * 8u) {
  const int64_t g = (n + per - 1) / per;
  return (unsigned)(g < 1 ? 1 : (g > cap ? cap : g));
}

}  // namespace

hipError_t launch_sample(const int32_t *ids, const int64_t *off, const int32_t *coe,
                         const int32_t *labels, int32_t *idx, int32_t *y, int32_t *hits, int C,
                         int B, int K, uint64_t seed, int64_t step0, int nsteps, int64_t max_steps,
                         hipStream_t s) {
  hipLaunchKernelGGL(sample_kernel, dim3(C, nsteps), dim3(256), 0, s, ids, off, coe, labels, idx, y,
                     hits, C, B, K, seed, step0, max_steps);
  return hipGetLastError();
}

hipError_t launch_gather(const float *images, const int32_t *idx, void *x, int dtype, int64_t rows,
                         int64_t row_elems, hipStream_t s) {
  if (dtype == GCPSL_BF16)
    hipLaunchKernelGGL(gather_kernel<bf16_t>, dim3((unsigned)rows), dim3(256), 0, s, images, idx,
                       (bf16_t *)x, row_elems);
  else
    hipLaunchKernelGGL(gather_kernel<float>, dim3((unsigned)rows), dim3(256), 0, s, images, idx,
                       (float *)x, row_elems);
  return hipGetLastError();
}

hipError_t launch_gather_im2col(const float *images, const int32_t *idx, void *x, int dtype, int64_t rows,
                                int H, int W, int Cin, int Kc, hipStream_t s) {
  const size_t img = sizeof(float) * (size_t)H * W * Cin;
  const int use_lds = img <= 64 * 1024 ? 1 : 0;
  const size_t shm = use_lds ? img : 0;
  if (dtype == GCPSL_BF16)
    hipLaunchKernelGGL(gather_im2col_kernel<bf16_t>, dim3((unsigned)rows), dim3(256), shm, s, images, idx,
                       (bf16_t *)x, H, W, Cin, Kc, use_lds);
  else
    hipLaunchKernelGGL(gather_im2col_kernel<float>, dim3((unsigned)rows), dim3(256), shm, s, images, idx,
                       (float *)x, H, W, Cin, Kc, use_lds);
  return hipGetLastError();
}

hipError_t launch_prep_weights(int dtype, const float *theta, int64_t P, int C, int64_t w_off,
                               int co, int ci, void *wf, int Kp, void *wd, int Kdp, hipStream_t s) {
  const dim3 grid(grid_for((int64_t)co * Kp, 256, 4096), C);
  const dim3 gridd(((co + 63) / 64) * ((ci + 63) / 64), 9, C);
  if (dtype == GCPSL_BF16) {
    hipLaunchKernelGGL(prep_wf_kernel<bf16_t>, grid, dim3(256), 0, s, theta, P, w_off, co, ci,
                       (bf16_t *)wf, Kp);
    if (wd)
      hipLaunchKernelGGL(prep_wd_kernel<bf16_t>, gridd, dim3(256), 0, s, theta, P, w_off, co, ci,
                         (bf16_t *)wd, Kdp);
  } else {
    hipLaunchKernelGGL(prep_wf_kernel<float>, grid, dim3(256), 0, s, theta, P, w_off, co, ci,
                       (float *)wf, Kp);
    if (wd)
      hipLaunchKernelGGL(prep_wd_kernel<float>, gridd, dim3(256), 0, s, theta, P, w_off, co, ci,
                         (float *)wd, Kdp);
  }
  return hipGetLastError();
}

hipError_t launch_maxpool_fwd(int dtype, const void *x, void *z, int C, int Bt, int H, int W, int Ch,
                              hipStream_t s) {
  const int64_t total = (int64_t)C * Bt * (H / 2) * (W / 2) * Ch;
  if (dtype == GCPSL_BF16)
    hipLaunchKernelGGL(maxpool_fwd_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const bf16_t *)x, (bf16_t *)z, total, H, W, Ch);
  else
    hipLaunchKernelGGL(maxpool_fwd_kernel<float>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const float *)x, (float *)z, total, H, W, Ch);
  return hipGetLastError();
}

hipError_t launch_maxpool_bwd(int dtype, const void *a, const void *gz, void *gpre, int C, int Bt,
                              int H, int W, int Ch, hipStream_t s) {
  const int64_t total = (int64_t)C * Bt * (H / 2) * (W / 2) * Ch;
  if (dtype == GCPSL_BF16)
    hipLaunchKernelGGL(maxpool_bwd_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const bf16_t *)a, (const bf16_t *)gz, (bf16_t *)gpre, total, H, W, Ch);
  else
    hipLaunchKernelGGL(maxpool_bwd_kernel<float>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const float *)a, (const float *)gz, (float *)gpre, total, H, W, Ch);
  return hipGetLastError();
}

hipError_t launch_head_pool(int dtype, const void *a, void *h, int C, int Bt, int H, int W, int Ch,
                            int maxpool, hipStream_t s) {
  const int64_t total = (int64_t)C * Bt * Ch;
  if (dtype == GCPSL_BF16)
    hipLaunchKernelGGL(head_pool_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const bf16_t *)a, (bf16_t *)h, total, H, W, Ch, maxpool);
  else
    hipLaunchKernelGGL(head_pool_kernel<float>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const float *)a, (float *)h, total, H, W, Ch, maxpool);
  return hipGetLastError();
}

hipError_t launch_linear_ce(int dtype, const void *h, const int32_t *y, const float *theta, int64_t P,
                            int64_t w_off, int64_t b_off, float *grad, float *dh, float *loss, int C,
                            int Bt, int Ch, int L, hipStream_t s) {
  const size_t shm = linear_ce_lds_bytes(Bt, Ch, L);
  if (shm > kMaxLinearLds) return hipErrorInvalidValue;
  if (shm > 64 * 1024) {
    const hipError_t e = dtype == GCPSL_BF16
        ? hipFuncSetAttribute(reinterpret_cast<const void *>(linear_ce_kernel<bf16_t>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm)
        : hipFuncSetAttribute(reinterpret_cast<const void *>(linear_ce_kernel<float>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    if (e != hipSuccess) return e;
  }
  if (dtype == GCPSL_BF16)
    hipLaunchKernelGGL(linear_ce_kernel<bf16_t>, dim3(C), dim3(1024), shm, s, (const bf16_t *)h, y,
                       theta, P, w_off, b_off, grad, dh, loss, Bt, Ch, L);
  else
    hipLaunchKernelGGL(linear_ce_kernel<float>, dim3(C), dim3(1024), shm, s, (const float *)h, y,
                       theta, P, w_off, b_off, grad, dh, loss, Bt, Ch, L);
  return hipGetLastError();
}

hipError_t launch_head_pool_bwd(int dtype, const void *a, const float *dh, void *gpre, int C, int Bt,
                                int H, int W, int Ch, int maxpool, hipStream_t s) {
  const int64_t total = maxpool ? (int64_t)C * Bt * (H / 2) * (W / 2) * Ch : (int64_t)C * Bt * H * W * Ch;
  if (dtype == GCPSL_BF16)
    hipLaunchKernelGGL(head_pool_bwd_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const bf16_t *)a, dh, (bf16_t *)gpre, total, H, W, Ch, maxpool);
  else
    hipLaunchKernelGGL(head_pool_bwd_kernel<float>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const float *)a, dh, (float *)gpre, total, H, W, Ch, maxpool);
  return hipGetLastError();
}

hipError_t launch_wgrad_reduce(const float *dw, const float *db, int splits, int64_t dw_ss,
                               int64_t dw_rs, int64_t db_ss, int64_t db_rs, float *grad, int64_t P,
                               int64_t w_off, int64_t b_off, int64_t nw, int co, int C,
                               hipStream_t s) {
  hipLaunchKernelGGL(wgrad_reduce_kernel, dim3(grid_for(nw + co, 256, 4096), C), dim3(256), 0, s, dw,
                     db, splits, dw_ss, dw_rs, db_ss, db_rs, grad, P, w_off, b_off, nw, co);
  return hipGetLastError();
}

hipError_t launch_sgd(float *theta, float *mom, const float *grad, int64_t n, float lr, float mu,
                      hipStream_t s) {
  hipLaunchKernelGGL(sgd_kernel, dim3(grid_for(n / 4 + 1, 256, 8192)), dim3(256), 0, s, theta, mom,
                     grad, n, lr, mu);
  return hipGetLastError();
}

hipError_t launch_fuse(float *theta, const double *weights, double W, int C, int64_t P,
                       hipStream_t s) {
  hipLaunchKernelGGL(fuse_kernel, dim3(grid_for(P, 256, 8192)), dim3(256), 0, s, theta, weights, W, C,
                     P);
  return hipGetLastError();
}
