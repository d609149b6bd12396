// Sampling, gather, pools, the classifier head, SGD and fusion kernels.
#include <algorithm>

#include "rng.h"
#include "runtime.h"

namespace {

constexpr int kMaxBitmapWords = 2048;  // clients tracked per cluster: K <= 65536

// ---------------------------------------------------------------- sampling
// Eq. 1 / Eq. 3: cluster n's batch at its local round s is B distinct
// examples of its own pool: positions [tB, (t+1)B) of the keyed permutation
// of epoch e = s / S_n, t = s mod S_n, S_n = floor(n_n / B).  Also counts the
// distinct clients of the batch, |A_{n,t}| (Sec. III-A), and the batch
// deviation of Sec. V-E, the l1 distance between the batch's class
// distribution and the global one, as the exact integer numerator
// sum_c |h_c |D| - B g_c| (over B |D|; h_c: the batch's examples of class c,
// g_c: the data set's).
// Lockstep schedule (R = 0): every cluster takes its round s = step at every
// step.  Epoch-barrier schedule (R = max_n S_n slots per system epoch,
// Sec. III-A, Sec. IV-D): step = m R + t is slot t of system epoch m; cluster
// n takes its round m S_n + t (epoch m, position t) when t < S_n and waits
// otherwise -- no batch (ids and labels -1) and no participating client.
__global__ void __launch_bounds__(256)
sample_kernel(const int32_t *__restrict__ ids, const int64_t *__restrict__ off,
              const int32_t *__restrict__ coe, const int32_t *__restrict__ labels,
              const int64_t *__restrict__ ghist, int32_t *__restrict__ idx, int32_t *__restrict__ y,
              int32_t *__restrict__ hits, int64_t *__restrict__ dev, int C, int B, int K, int L, int64_t nex,
              uint64_t seed, int64_t step0, int64_t max_steps, int64_t R) {
  __shared__ uint32_t bitmap[kMaxBitmapWords];
  __shared__ int32_t hist[kMaxDevClasses];
  __shared__ int count;
  __shared__ unsigned long long dsum;
  const int n = blockIdx.x, j = blockIdx.y, tid = threadIdx.x;
  const int64_t step = step0 + j;
  const int64_t lo = off[n];
  const uint32_t nn = (uint32_t)(off[n + 1] - lo);
  const int64_t S = nn / (uint32_t)B;
  const int64_t e = R > 0 ? step / R : step / S, t = R > 0 ? step % R : step % S;
  if (t >= S) {  // waits at the epoch barrier
    for (int i = tid; i < B; i += blockDim.x) {
      const int64_t o = ((int64_t)j * C + n) * B + i;
      idx[o] = -1;
      y[o] = -1;
    }
    if (tid == 0 && step < max_steps) {
      hits[step * C + n] = 0;
      dev[step * C + n] = -1;  // no batch
    }
    return;
  }
  const uint64_t key = gc_sample_key(seed, (uint64_t)n, (uint64_t)e);
  const int words = (K + 31) >> 5;
  for (int w = tid; w < words; w += blockDim.x) bitmap[w] = 0u;
  for (int c = tid; c < L; c += blockDim.x) hist[c] = 0;
  if (tid == 0) {
    count = 0;
    dsum = 0ull;
  }
  __syncthreads();
  for (int i = tid; i < B; i += blockDim.x) {
    const uint32_t p = (uint32_t)(t * B + i);
    const int32_t ex = ids[lo + gc_permute(p, nn, key)];
    const int64_t o = ((int64_t)j * C + n) * B + i;
    const int32_t lab = labels[ex];
    idx[o] = ex;
    y[o] = lab;
    if ((uint32_t)lab < (uint32_t)L) atomicAdd(&hist[lab], 1);  // labels checked at create
    const int32_t c = coe[ex];
    atomicOr(&bitmap[c >> 5], 1u << (c & 31));
  }
  __syncthreads();
  int local = 0;
  for (int w = tid; w < words; w += blockDim.x) local += __popc(bitmap[w]);
  atomicAdd(&count, local);
  // |h_c |D| - B g_c| < 2^62 and their sum < 2^63: B |D| < 2^62 (B < 2^29, |D| < 2^31)
  unsigned long long dl = 0ull;
  for (int c = tid; c < L; c += blockDim.x) {
    const int64_t d = (int64_t)hist[c] * nex - (int64_t)B * ghist[c];
    dl += (unsigned long long)(d < 0 ? -d : d);
  }
  atomicAdd(&dsum, dl);
  __syncthreads();
  if (tid == 0 && step < max_steps) {
    hits[step * C + n] = count;
    dev[step * C + n] = (int64_t)dsum;
  }
}

template <typename T>
__global__ void __launch_bounds__(256)
gather_kernel(const float *__restrict__ images, const int32_t *__restrict__ idx, T *__restrict__ x,
              int64_t row_elems) {
  const int64_t row = blockIdx.x;
  if (idx[row] < 0) return;  // cluster waits at the epoch barrier
  const float *src = images + (int64_t)idx[row] * row_elems;
  T *dst = x + row * row_elems;
  if ((row_elems & 3) == 0) {
    const int64_t nv = row_elems >> 2;
    for (int64_t v = threadIdx.x; v < nv; v += blockDim.x) {
      const float4 f = reinterpret_cast<const float4 *>(src)[v];
      if constexpr (sizeof(T) == 4) {
        reinterpret_cast<float4 *>(dst)[v] = f;
      } else {
        const uint32_t lo = pack2_bf16(f.x, f.y);
        const uint32_t hi = pack2_bf16(f.z, f.w);
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
  if (idx[row] < 0) return;  // cluster waits at the epoch barrier
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

// The same staging for a compile-time channel count CIN and row width KC
// (the 3-channel image layer).  The image sits in LDS with a one-pixel zero
// border, so no tap needs a bounds test.  A workgroup stages several
// examples in turn: while it writes the rows of one example from LDS, the
// 16-byte loads of the next example's image (NV4 per thread) are already in
// flight.  A thread always fills the same VEC-column chunk of a row (the
// thread count is a multiple of the chunks per row), so its VEC source
// offsets are computed once; lanes of a wave write consecutive 16-byte chunks
// of consecutive pixels.
template <typename T, int CIN, int KC, int NV4>
__global__ void __launch_bounds__(256)
gather_im2col_fixed_kernel(const float *__restrict__ images, const int32_t *__restrict__ idx,
                           T *__restrict__ x, int H, int W, FastDiv fd_w, int64_t rows, int per_wg) {
  extern __shared__ float img[];  // [(H + 2) * (W + 2) * CIN]
  constexpr int VEC = ElemT<T>::VEC, NCH = KC / VEC;
  static_assert(KC % VEC == 0 && KC >= 9 * CIN, "row width");
  const int nthr = (blockDim.x / NCH) * NCH;
  const int tid = threadIdx.x;
  const int Wp = W + 2, npad = (H + 2) * Wp * CIN, n4 = H * W * CIN / 4;
  const int64_t r0 = (int64_t)blockIdx.x * per_wg;
  const int64_t r1 = min(rows, r0 + per_wg);
  for (int i = tid; i < npad; i += blockDim.x) img[i] = 0.f;  // the border stays zero
  const int j = tid % NCH;
  int off[VEC];  // source offsets; columns past 9 CIN read offset 0 and are zeroed
  uint32_t live = 0;
#pragma unroll
  for (int e = 0; e < VEC; ++e) {
    const int k = j * VEC + e;
    const int rs = k / CIN, c = k - rs * CIN;
    off[e] = k < 9 * CIN ? ((rs / 3) * Wp + rs % 3) * CIN + c : 0;
    live |= (k < 9 * CIN ? 1u : 0u) << e;
  }
  // LDS destinations of this thread's staged image values and its first
  // output pixel: the same for every example, so computed once
  int sdst[NV4][4];
#pragma unroll
  for (int u = 0; u < NV4; ++u)
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int i = 4 * (tid + u * 256) + t;
      const int q = i / CIN, c = i - q * CIN;
      const int h = (int)fdiv((uint32_t)q, fd_w), w = q - h * W;
      sdst[u][t] = ((h + 1) * Wp + w + 1) * CIN + c;
    }
  const int pstep = nthr / NCH;  // pixels per pass of the workgroup
  const int sh = (int)fdiv((uint32_t)pstep, fd_w), sw = pstep - sh * W;
  const int p0 = tid / NCH;
  const int h0 = (int)fdiv((uint32_t)p0, fd_w), w0 = p0 - h0 * W;
  float4 pre[NV4];
  auto fetch = [&](int64_t row) {
    const float4 *src = reinterpret_cast<const float4 *>(images + (int64_t)idx[row] * (4 * n4));
#pragma unroll
    for (int u = 0; u < NV4; ++u) {
      const int v = tid + u * 256;
      if (v < n4) pre[u] = src[v];
    }
  };
  // rows without a batch (a cluster waiting at the epoch barrier) are skipped
  if (r0 < r1 && idx[r0] >= 0) fetch(r0);
  for (int64_t row = r0; row < r1; ++row) {
    const bool has_batch = idx[row] >= 0;
    __syncthreads();  // the previous example's reads of LDS are done
#pragma unroll
    for (int u = 0; u < NV4; ++u) {
      const int v = tid + u * 256;
      if (has_batch && v < n4) {
        const float f[4] = {pre[u].x, pre[u].y, pre[u].z, pre[u].w};
#pragma unroll
        for (int t = 0; t < 4; ++t) img[sdst[u][t]] = f[t];
      }
    }
    __syncthreads();
    if (row + 1 < r1 && idx[row + 1] >= 0) fetch(row + 1);
    if (has_batch && tid < nthr) {
      T *dst = x + row * (int64_t)H * W * KC + j * VEC;
      int h = h0, w = w0;  // pixel p = h W + w, advanced by pstep per pass
      for (int p = p0; p < H * W; p += pstep) {
        const float *base = img + (h * Wp + w) * CIN;
        w += sw;
        h += sh + (w >= W ? 1 : 0);
        w -= w >= W ? W : 0;
        struct { T v[VEC]; } pk;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const float v = base[off[e]];
          pk.v[e] = ElemT<T>::from_f(((live >> e) & 1u) ? v : 0.f);
        }
        // streaming store: the rows are written once and read by the next
        // kernel, they need no cache allocation on the way out
        typedef unsigned U4 __attribute__((ext_vector_type(4)));
        __builtin_nontemporal_store(__builtin_bit_cast(U4, pk), reinterpret_cast<U4 *>(dst + (int64_t)p * KC));
      }
    }
  }
}

// ------------------------------------------------------ weight preparation
// Compute copies of the conv layers' weights from the fp32 masters:
//   wf[co][k], k = (r, s, ci) < 9 ci, rows zero-padded to Kp (forward);
//   wd[ci][kk], kk = (r', s', co), wd[ci][(r', s', co)] = W[co][2-r'][2-s'][ci]
//   rows zero-padded to Kdp (input gradient as a forward conv).
// wf is a row copy; wd is a transpose of 64 x 64 (co, ci) blocks per kernel
// tap, staged through LDS so both the reads and the writes are coalesced.
// One launch covers every layer: workgroup b belongs to the job whose first
// workgroup is the largest not above b.
// Eight consecutive outputs from fp32 values: one 16-byte store for bf16,
// two for fp32 (p is 8-element aligned).
template <typename T>
__device__ __forceinline__ void store8(T *p, const float (&v)[8]) {
  if constexpr (sizeof(T) == 2) {
    uint4 o;
    o.x = pack2_bf16(v[0], v[1]);
    o.y = pack2_bf16(v[2], v[3]);
    o.z = pack2_bf16(v[4], v[5]);
    o.w = pack2_bf16(v[6], v[7]);
    *reinterpret_cast<uint4 *>(p) = o;
  } else {
    *reinterpret_cast<float4 *>(p) = make_float4(v[0], v[1], v[2], v[3]);
    *reinterpret_cast<float4 *>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
  }
}

// Both copies of one 64 x 64 (co, ci) block of source tap ts = (r, s): the
// block is read once into LDS, written to wf at tap ts (rows co) and,
// transposed, to wd at the flipped tap 8 - ts (rows ci).  co and ci are
// multiples of 8, so every 8-element run is wholly inside or outside the
// layer and 16-byte aligned (Kp, Kdp are multiples of 8 as well).  The
// workgroups of tap 0 also zero the row padding of their blocks.
template <typename T>
__device__ __forceinline__ void prep_both_block(const float *w, int rep, const PrepJob &J, int lb,
                                                float (&tile)[64][65]) {
  const int co = J.co, ci = J.ci, K = 9 * ci, Kdp = J.kpad, Kp = J.kpad2;
  const int nco = (co + 63) / 64;
  const int ts = lb % 9, blk = lb / 9;
  const int cb = blk % nco, ib = blk / nco;
  const int tid = threadIdx.x, tx = tid & 63, ty = tid >> 6;
  float v[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int o = cb * 64 + ty + 4 * i, c = ib * 64 + tx;
    v[i] = (o < co && c < ci) ? w[(int64_t)o * K + ts * ci + c] : 0.f;
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) tile[ty + 4 * i][tx] = v[i];
  __syncthreads();
  T *wf = reinterpret_cast<T *>(J.dst2) + (int64_t)rep * co * Kp;
  T *wd = reinterpret_cast<T *>(J.dst) + (int64_t)rep * ci * Kdp;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int q = tid + 256 * k, r = q >> 3, run = 8 * (q & 7);
    // forward copy: row o = cb 64 + r, columns ts ci + ib 64 + run ..
    const int o = cb * 64 + r, c = ib * 64 + run;
    if (o < co && c < ci) {
      float e[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) e[t] = tile[r][run + t];
      store8(wf + (int64_t)o * Kp + ts * ci + c, e);
    }
    // input-gradient copy: row c = ib 64 + r, columns (8 - ts) co + cb 64 + run ..
    const int c2 = ib * 64 + r, o2 = cb * 64 + run;
    if (c2 < ci && o2 < co) {
      float e[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) e[t] = tile[run + t][r];
      store8(wd + (int64_t)c2 * Kdp + (8 - ts) * co + o2, e);
    }
  }
  if (ts == 0) {
    const float z[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (ib == 0) {  // wf columns 9 ci .. Kp of this block's rows
      const int runs = (Kp - K) / 8;
      for (int q = tid; q < 64 * runs; q += 256) {
        const int o = cb * 64 + q / runs;
        if (o < co) store8(wf + (int64_t)o * Kp + K + 8 * (q % runs), z);
      }
    }
    if (cb == 0) {  // wd columns 9 co .. Kdp of this block's rows
      const int runs = (Kdp - 9 * co) / 8;
      for (int q = tid; q < 64 * runs; q += 256) {
        const int c = ib * 64 + q / runs;
        if (c < ci) store8(wd + (int64_t)c * Kdp + 9 * co + 8 * (q % runs), z);
      }
    }
  }
}

template <typename T>
__global__ void __launch_bounds__(256)
prep_weights_kernel(const float *__restrict__ theta, const int32_t *__restrict__ rmap, int64_t P, PrepJobs jobs) {
  __shared__ float tile[64][65];
  const int b = blockIdx.x;
  int jn = 0;
  while (jn + 1 < jobs.n && jobs.j[jn + 1].first <= b) ++jn;
  const PrepJob &J = jobs.j[jn];
  const int rep = replica_of(rmap, blockIdx.y);
  const float *w = theta + rep * P + J.w_off;
  const int co = J.co, ci = J.ci, taps = J.taps, K = taps * ci;
  const int lb = b - J.first;
  if (J.kind == 0) {
    // forward copy: output row lb
    T *dst = reinterpret_cast<T *>(J.dst) + ((int64_t)rep * co + lb) * J.kpad;
    const float *src = w + (int64_t)lb * K;
    // 8 consecutive outputs per thread: 8 independent loads (the source row
    // need not be vector-aligned), one 16-byte store per 16 output bytes
    // (kpad is a multiple of the 32- or 64-wide k tile, so every run is
    // aligned and inside the row)
    for (int k0 = threadIdx.x * 8; k0 < J.kpad; k0 += blockDim.x * 8) {
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = k0 + e < K ? src[k0 + e] : 0.f;
      if constexpr (sizeof(T) == 2) {
        uint4 o;
        o.x = pack2_bf16(v[0], v[1]);
        o.y = pack2_bf16(v[2], v[3]);
        o.z = pack2_bf16(v[4], v[5]);
        o.w = pack2_bf16(v[6], v[7]);
        *reinterpret_cast<uint4 *>(dst + k0) = o;
      } else {
        *reinterpret_cast<float4 *>(dst + k0) = make_float4(v[0], v[1], v[2], v[3]);
        *reinterpret_cast<float4 *>(dst + k0 + 4) = make_float4(v[4], v[5], v[6], v[7]);
      }
    }
    return;
  }
  if (J.kind == 2) {
    prep_both_block<T>(w, rep, J, lb, tile);
    return;
  }
  // input-gradient copy: block (cb, ib) of tap `tap` of the flipped kernel
  // (one tap: the transpose)
  const int Kdp = J.kpad;
  const int nco = (co + 63) / 64;
  const int tap = lb % taps, blk = lb / taps;
  const int cb = blk % nco, ib = blk / nco;
  const int rs_src = taps - 1 - tap;  // (2 - r') * 3 + (2 - s')
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  // 16 rows per thread with every load in flight (fixed trip counts)
  float v[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int r = ty + 4 * i, o = cb * 64 + r, c = ib * 64 + tx;
    v[i] = (o < co && c < ci) ? w[(int64_t)o * K + rs_src * ci + c] : 0.f;
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) tile[ty + 4 * i][tx] = v[i];
  __syncthreads();
  T *dst = reinterpret_cast<T *>(J.dst) + (int64_t)rep * ci * Kdp;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int r = ty + 4 * i, c = ib * 64 + r, o = cb * 64 + tx;
    if (c < ci && o < co) dst[(int64_t)c * Kdp + tap * co + o] = ElemT<T>::from_f(tile[tx][r]);
  }
  // zero the row padding once per row (by the first tap/co block)
  if (tap == 0 && cb == 0) {
    for (int r = ty; r < 64; r += 4) {
      const int c = ib * 64 + r;
      if (c >= ci) continue;
      for (int k = taps * co + tx; k < Kdp; k += 64) dst[(int64_t)c * Kdp + k] = T(0);
    }
  }
}

// -------------------------------------------------------------- max pool
// 2x2 / stride 2 over a [N][H][W][Ch] batch (N examples).  The backward pass
// routes each pooled gradient to the first maximum of its window in
// row-major order (strict >) and applies the producing conv's ReLU mask
// (output > 0).  A thread handles one 16-byte vector of VEC channels of one
// output position; index arithmetic within a replica is 32-bit.

// One 16-byte vector of activations.
template <typename T> struct Vec16 {
  T v[ElemT<T>::VEC];
};
template <typename T>
__device__ __forceinline__ Vec16<T> ld16(const T *p) {
  return __builtin_bit_cast(Vec16<T>, *reinterpret_cast<const uint4 *>(p));
}
template <typename T>
__device__ __forceinline__ void st16(T *p, const Vec16<T> &v) {
  *reinterpret_cast<uint4 *>(p) = __builtin_bit_cast(uint4, v);
}

// Output vector i of a pooled [N][Ho][Wo][CV] grid -> offset of the top-left
// input element of its window, the example and the channel vector.
struct PoolIdx {
  FastDiv cv, wo, ho;
};
__device__ __forceinline__ int64_t pool_base(uint32_t i, const PoolIdx &d, int W, int Ch, int VEC, uint32_t *bi,
                                             int *cv) {
  const uint32_t r = fdiv(i, d.cv);
  *cv = (int)(i - r * d.cv.d);
  const uint32_t r2 = fdiv(r, d.wo);
  const int wo = (int)(r - r2 * d.wo.d);
  *bi = fdiv(r2, d.ho);
  const int ho = (int)(r2 - *bi * d.ho.d);
  return (((int64_t)*bi * (2 * d.ho.d) + 2 * ho) * W + 2 * wo) * Ch + *cv * VEC;
}

template <typename T>
__global__ void __launch_bounds__(256)
maxpool_fwd_kernel(const T *__restrict__ x, T *__restrict__ z, const int32_t *__restrict__ rmap, int64_t x_rs,
                   int64_t z_rs, uint32_t total, PoolIdx d, int W, int Ch) {
  constexpr int VEC = ElemT<T>::VEC;
  const uint32_t i = blockIdx.x * 256u + threadIdx.x;
  if (i >= total) return;
  const int rep = replica_of(rmap, blockIdx.y);
  x += rep * x_rs;
  z += rep * z_rs;
  uint32_t bi;
  int cv;
  const int64_t base = pool_base(i, d, W, Ch, VEC, &bi, &cv);
  const Vec16<T> q[4] = {ld16(x + base), ld16(x + base + Ch), ld16(x + base + (int64_t)W * Ch),
                         ld16(x + base + (int64_t)W * Ch + Ch)};
  Vec16<T> out;
#pragma unroll
  for (int e = 0; e < VEC; ++e) {
    float m = ElemT<T>::to_f(q[0].v[e]);
    T best = q[0].v[e];
#pragma unroll
    for (int k = 1; k < 4; ++k) {
      const float v = ElemT<T>::to_f(q[k].v[e]);
      if (v > m) {
        m = v;
        best = q[k].v[e];
      }
    }
    out.v[e] = best;
  }
  st16(z + (int64_t)i * VEC, out);
}

// gpre over the window of output vector i: the gradient g[e] goes to the
// first maximum of a (if it is > 0), zero elsewhere.
template <typename T>
__device__ __forceinline__ void route_window(const T *__restrict__ a, T *__restrict__ gpre, int64_t base, int W,
                                             int Ch, const Vec16<T> &g) {
  constexpr int VEC = ElemT<T>::VEC;
  const int64_t o[4] = {base, base + Ch, base + (int64_t)W * Ch, base + (int64_t)W * Ch + Ch};
  Vec16<T> q[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) q[k] = ld16(a + o[k]);
  Vec16<T> out[4];
#pragma unroll
  for (int e = 0; e < VEC; ++e) {
    float v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = ElemT<T>::to_f(q[k].v[e]);
    int arg = 0;
#pragma unroll
    for (int k = 1; k < 4; ++k)
      if (v[k] > v[arg]) arg = k;
#pragma unroll
    for (int k = 0; k < 4; ++k) out[k].v[e] = (k == arg && v[k] > 0.f) ? g.v[e] : T(0);
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) st16(gpre + o[k], out[k]);
}

template <typename T>
__global__ void __launch_bounds__(256)
maxpool_bwd_kernel(const T *__restrict__ a, const T *__restrict__ gz, T *__restrict__ gpre,
                   const int32_t *__restrict__ rmap, int64_t a_rs, int64_t z_rs, uint32_t total, PoolIdx d, int W,
                   int Ch) {
  constexpr int VEC = ElemT<T>::VEC;
  const uint32_t i = blockIdx.x * 256u + threadIdx.x;
  if (i >= total) return;
  const int rep = replica_of(rmap, blockIdx.y);
  a += rep * a_rs;
  gpre += rep * a_rs;
  gz += rep * z_rs;
  uint32_t bi;
  int cv;
  const int64_t base = pool_base(i, d, W, Ch, VEC, &bi, &cv);
  route_window(a, gpre, base, W, Ch, ld16(gz + (int64_t)i * VEC));
}

// ------------------------------------------------------------------ head
// Pooled feature h[n][c] = mean over positions of the (optionally 2x2 max
// pooled) last conv output.  One workgroup per (example, block of CVB
// channel vectors); the positions are split over G = 256 / CVB thread groups
// whose fp32 partial sums are added in group order.
template <typename T>
__global__ void __launch_bounds__(256)
head_pool_kernel(const T *__restrict__ a, T *__restrict__ h, const int32_t *__restrict__ rmap, int Bt, int H, int W,
                 int Ch, int CVB, int maxpool) {
  constexpr int VEC = ElemT<T>::VEC;
  __shared__ float part[256 * VEC];
  const int64_t bi = (int64_t)replica_of(rmap, blockIdx.z) * Bt + blockIdx.x;
  const int tid = threadIdx.x;
  const int G = 256 / CVB;
  const int cvl = tid % CVB, g = tid / CVB;
  const int cv = blockIdx.y * CVB + cvl;
  const int CV = Ch / VEC;
  const T *src = a + (int64_t)bi * H * W * Ch + cv * VEC;
  const int Wo = maxpool ? W / 2 : W, npos = maxpool ? (H / 2) * (W / 2) : H * W;
  float sum[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) sum[e] = 0.f;
  if (g < G && cv < CV) {
    for (int q = g; q < npos; q += G) {
      const int ho = q / Wo, wo = q - ho * Wo;
      if (maxpool) {
        const int64_t b0 = ((int64_t)(2 * ho) * W + 2 * wo) * Ch;
        const Vec16<T> v0 = ld16(src + b0), v1 = ld16(src + b0 + Ch), v2 = ld16(src + b0 + (int64_t)W * Ch),
                       v3 = ld16(src + b0 + (int64_t)W * Ch + Ch);
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          float m = ElemT<T>::to_f(v0.v[e]);
          m = fmaxf(m, ElemT<T>::to_f(v1.v[e]));
          m = fmaxf(m, ElemT<T>::to_f(v2.v[e]));
          m = fmaxf(m, ElemT<T>::to_f(v3.v[e]));
          sum[e] += m;
        }
      } else {
        const Vec16<T> v = ld16(src + ((int64_t)ho * W + wo) * Ch);
#pragma unroll
        for (int e = 0; e < VEC; ++e) sum[e] += ElemT<T>::to_f(v.v[e]);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < VEC; ++e) part[tid * VEC + e] = sum[e];
  __syncthreads();
  if (tid < CVB && cv < CV) {
    Vec16<T> out;
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      float s = 0.f;
      for (int k = 0; k < G; ++k) s += part[(k * CVB + tid) * VEC + e];
      out.v[e] = ElemT<T>::from_f(s / (float)npos);
    }
    st16(h + (int64_t)bi * Ch + cv * VEC, out);
  }
}

// Linear layer and mean softmax cross-entropy for one replica per workgroup:
// logits = h W^T + b; with label smoothing eps (Sec. V-A) the target is
// q = (1 - eps) onehot(y) + eps / L, loss = mean_b -sum_j q_j log softmax_j,
// dlogits = (softmax - q) / B, dW = dlogits^T h, db = sum_b dlogits,
// dh = dlogits W.  bf16 workloads use the bf16-rounded weight matrix.  The
// pooled features, the weights and the logits are staged in LDS so every
// global access is coalesced; each sum runs in a fixed order.
template <typename T>
__global__ void __launch_bounds__(1024)
linear_ce_kernel(const T *__restrict__ h, const int32_t *__restrict__ y,
                 const float *__restrict__ theta, int64_t P, int64_t w_off, int64_t b_off,
                 float *__restrict__ grad, float *__restrict__ dh, float *__restrict__ loss,
                 const int32_t *__restrict__ rmap, int Bt, int Ch, int L, float eps) {
  extern __shared__ float sh[];
  // rows padded to Ch + 1 floats: threads of a wave that read the same
  // column of different rows hit different banks
  const int CP = Ch + 1;
  float *hs = sh;                      // [Bt][CP]
  float *ws = hs + (int64_t)Bt * CP;   // [L][CP]
  float *lg = ws + (int64_t)L * CP;    // [Bt][L] logits, then dlogits
  float *lossb = lg + Bt * L;          // [Bt]
  float *bs = lossb + Bt;              // [L] bias
  const int rep = replica_of(rmap, blockIdx.x), tid = threadIdx.x, nt = blockDim.x;
  const T *hr = h + (int64_t)rep * Bt * Ch;
  const float *Wl = theta + rep * P + w_off;
  const float *bl = theta + rep * P + b_off;
  // staging: whole 16-byte vectors when rows hold them, several loads in
  // flight per thread (the loop is latency-bound otherwise)
  constexpr int V = ElemT<T>::VEC;
  if (Ch % V == 0) {
    const int nv = Bt * Ch / V;
#pragma unroll 4
    for (int i = tid; i < nv; i += nt) {
      const uint4 u = reinterpret_cast<const uint4 *>(hr)[i];
      const T *e = reinterpret_cast<const T *>(&u);
      const int b = (i * V) / Ch, c = (i * V) % Ch;
#pragma unroll
      for (int k = 0; k < V; ++k) hs[b * CP + c + k] = ElemT<T>::to_f(e[k]);
    }
  } else {
    for (int i = tid; i < Bt * Ch; i += nt) hs[(i / Ch) * CP + i % Ch] = ElemT<T>::to_f(hr[i]);
  }
#pragma unroll 4
  for (int i = tid; i < L * Ch; i += nt) ws[(i / Ch) * CP + i % Ch] = ElemT<T>::to_f(ElemT<T>::from_f(Wl[i]));
  for (int j = tid; j < L; j += nt) bs[j] = bl[j];
  __syncthreads();
  for (int i = tid; i < Bt * L; i += nt) {
    const int b = i / L, j = i % L;
    const float *hb = hs + (int64_t)b * CP, *wj = ws + (int64_t)j * CP;
    // two partial sums over unrolled runs keep several LDS reads in flight
    float s0 = 0.f, s1 = 0.f;
    int c = 0;
#pragma unroll 4
    for (; c + 1 < Ch; c += 2) {
      s0 += hb[c] * wj[c];
      s1 += hb[c + 1] * wj[c + 1];
    }
    if (c < Ch) s0 += hb[c] * wj[c];
    float s = bs[j] + (s0 + s1);
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
    // target q = (1 - eps) onehot(y) + eps / L; loss -sum_j q_j log p_j
    const float qo = eps / (float)L, qy = 1.f - eps + qo;
    float zs = 0.f;
    for (int j = 0; j < L; ++j) zs += lg[b * L + j] - m;
    lossb[b] = eps > 0.f ? lse - (1.f - eps) * (lg[b * L + yb] - m) - qo * zs : lse - (lg[b * L + yb] - m);
    for (int j = 0; j < L; ++j) {
      const float p = expf(lg[b * L + j] - m - lse);
      lg[b * L + j] = (p - (j == yb ? qy : qo)) / (float)Bt;
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
    float s0 = 0.f, s1 = 0.f;
    int b = 0;
#pragma unroll 4
    for (; b + 1 < Bt; b += 2) {
      s0 += lg[b * L + j] * hs[(int64_t)b * CP + c];
      s1 += lg[(b + 1) * L + j] * hs[(int64_t)(b + 1) * CP + c];
    }
    if (b < Bt) s0 += lg[b * L + j] * hs[(int64_t)b * CP + c];
    g[w_off + i] = s0 + s1;
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
#pragma unroll 4
    for (int j = 0; j < L; ++j) s += lg[b * L + j] * ws[(int64_t)j * CP + c];
    dhr[i] = s;
  }
}

// The same head with the weights in registers, for heads of at most 256
// channels and kHeadRegL classes: lane l of each wave holds channels
// 4l..4l+3 of every weight row (bf16-rounded for bf16 workloads), and wave w
// takes examples w, w + 8, ...  A lane forms its 4-channel share of every
// logit of an example; a butterfly over the 64 lanes adds the shares.  The
// input gradient of an example comes from the lane's own weights; the
// weight gradient is summed per wave over its examples, then over the
// waves in a fixed tree.  Every sum runs in a fixed order.  LM is L rounded
// up to a multiple of 4 (classes past L have zero weights and gradients).
// Loads never sit behind a branch: out-of-range lanes read a clamped,
// valid address and select zero, so every load of a group is in flight
// together.

// Channels c..c+3 of one example as floats.
template <typename T>
__device__ __forceinline__ void head_load4(const T *p, float x[4]) {
  if constexpr (sizeof(T) == 2) {
    const uint2 u = *reinterpret_cast<const uint2 *>(p);
    x[0] = __uint_as_float(u.x << 16);
    x[1] = __uint_as_float(u.x & 0xffff0000u);
    x[2] = __uint_as_float(u.y << 16);
    x[3] = __uint_as_float(u.y & 0xffff0000u);
  } else {
    const float4 f = *reinterpret_cast<const float4 *>(p);
    x[0] = f.x; x[1] = f.y; x[2] = f.z; x[3] = f.w;
  }
}

// One halving exchange over lane bit 2 N, for each of NB vectors at once
// (their exchanges are independent and overlap): a lane keeps half N / 2..
// of its N entries if that bit is set, else half 0.., and adds its
// partner's copy of the half it keeps.  A compile-time stage, so every
// index is a register.
template <int N, int NB>
__device__ __forceinline__ void wave_halve(float (&v)[NB][kHeadRegL], int lane) {
  const bool up = lane & (2 * N);
  float keep[NB][N / 2], got[NB][N / 2];
#pragma unroll
  for (int u = 0; u < NB; ++u)
#pragma unroll
    for (int i = 0; i < N / 2; ++i) {
      const float lo = v[u][i], hi = v[u][i + N / 2];  // both in registers, then a select
      keep[u][i] = up ? hi : lo;
      got[u][i] = __shfl_xor(up ? lo : hi, 2 * N, 64);
    }
#pragma unroll
  for (int u = 0; u < NB; ++u)
#pragma unroll
    for (int i = 0; i < N / 2; ++i) v[u][i] = keep[u][i] + got[u][i];
}

// Sums each of NB vectors v[u][0..15] over the 64 lanes of a wave: four
// halving exchanges leave entry (lane >> 2) & 15 in each lane, two more add
// the four lanes that hold the same entry (all four get the same value).
template <int NB>
__device__ __forceinline__ void wave_sum16(float (&v)[NB][kHeadRegL], float (&sum)[NB]) {
  static_assert(kHeadRegL == 16, "four halving stages");
  const int lane = threadIdx.x & 63;
  wave_halve<16>(v, lane);
  wave_halve<8>(v, lane);
  wave_halve<4>(v, lane);
  wave_halve<2>(v, lane);
  float t[NB];
#pragma unroll
  for (int u = 0; u < NB; ++u) t[u] = __shfl_xor(v[u][0], 2, 64);
#pragma unroll
  for (int u = 0; u < NB; ++u) sum[u] = v[u][0] + t[u];
#pragma unroll
  for (int u = 0; u < NB; ++u) t[u] = __shfl_xor(sum[u], 1, 64);
#pragma unroll
  for (int u = 0; u < NB; ++u) sum[u] += t[u];
}

template <typename T, int LM>
__global__ void __launch_bounds__(kHeadRegWaves * 64)
linear_ce_reg_kernel(const T *__restrict__ h, const int32_t *__restrict__ y,
                     const float *__restrict__ theta, int64_t P, int64_t w_off, int64_t b_off,
                     float *__restrict__ grad, float *__restrict__ dh, float *__restrict__ loss,
                     const int32_t *__restrict__ rmap, int Bt, int Ch, int L, float eps) {
  static_assert(LM % 4 == 0 && LM <= kHeadRegL, "class slots");
  constexpr int NW = kHeadRegWaves, NB = 4;  // NB examples' loads in flight per wave
  extern __shared__ float sh[];
  float *lg = sh;               // [Bt][L] logits, then dlogits
  float *lossb = lg + Bt * L;   // [Bt]
  float4 *red = reinterpret_cast<float4 *>(sh + ((Bt * (L + 1) + 3) & ~3));  // [NW / 2][L][64]
  const int rep = replica_of(rmap, blockIdx.x), tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int c0 = 4 * lane;
  const bool live = c0 < Ch;
  const int cl = live ? c0 : 0;  // a valid channel for every lane
  const T *hr = h + (int64_t)rep * Bt * Ch + cl;
  const float *Wl = theta + rep * P + w_off;
  const float *bl = theta + rep * P + b_off;
  float w[LM][4];
#pragma unroll
  for (int j = 0; j < LM; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float v = Wl[(int64_t)min(j, L - 1) * Ch + cl + e];
      w[j][e] = (live && j < L) ? ElemT<T>::to_f(ElemT<T>::from_f(v)) : 0.f;
    }
  const int y0 = tid < Bt ? y[(int64_t)rep * Bt + tid] : 0;
  const int jl = (lane >> 2) & (kHeadRegL - 1);  // the logit this lane's sum ends as
  const bool writer = (lane & 3) == 0 && jl < L;
  const float bias = bl[min(jl, L - 1)];

  // logits; each group of NB examples issues the next group's loads first
  // (clamped to the last example past the end)
  float xn[NB][4];
#pragma unroll
  for (int u = 0; u < NB; ++u) head_load4(hr + (int64_t)min(wave + u * NW, Bt - 1) * Ch, xn[u]);
  for (int b0 = wave; b0 < Bt; b0 += NB * NW) {
    float x[NB][4];
#pragma unroll
    for (int u = 0; u < NB; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) x[u][e] = xn[u][e];
#pragma unroll
    for (int u = 0; u < NB; ++u) head_load4(hr + (int64_t)min(b0 + (NB + u) * NW, Bt - 1) * Ch, xn[u]);
    float v[NB][kHeadRegL], sum[NB];
#pragma unroll
    for (int u = 0; u < NB; ++u)
#pragma unroll
      for (int j = 0; j < kHeadRegL; ++j)
        v[u][j] = j < LM ? fmaf(x[u][3], w[j][3], fmaf(x[u][2], w[j][2], fmaf(x[u][1], w[j][1], x[u][0] * w[j][0])))
                         : 0.f;
    wave_sum16(v, sum);
    if (writer) {
#pragma unroll
      for (int u = 0; u < NB; ++u)
        if (b0 + u * NW < Bt) lg[(b0 + u * NW) * L + jl] = bias + sum[u];
    }
  }
  __syncthreads();
  // softmax cross-entropy per example, as in linear_ce_kernel (the label of
  // the first example of each thread was loaded at the start)
  for (int b = tid; b < Bt; b += NW * 64) {
    float m = lg[b * L];
    for (int j = 1; j < L; ++j) m = fmaxf(m, lg[b * L + j]);
    float s = 0.f;
    for (int j = 0; j < L; ++j) s += expf(lg[b * L + j] - m);
    const float lse = logf(s);
    const int yb = b == tid ? y0 : y[(int64_t)rep * Bt + b];
    const float qo = eps / (float)L, qy = 1.f - eps + qo;
    float zs = 0.f;
    for (int j = 0; j < L; ++j) zs += lg[b * L + j] - m;
    lossb[b] = eps > 0.f ? lse - (1.f - eps) * (lg[b * L + yb] - m) - qo * zs : lse - (lg[b * L + yb] - m);
    for (int j = 0; j < L; ++j) {
      const float p = expf(lg[b * L + j] - m - lse);
      lg[b * L + j] = (p - (j == yb ? qy : qo)) / (float)Bt;
    }
  }
  __syncthreads();
  // the mean loss and the bias gradient: sums over the examples as 8
  // interleaved partial sums added in a fixed order (8 LDS reads in flight
  // instead of one), by the last wave, which has no more head work than
  // the others
  float *g = grad + rep * P;
  if (wave == NW - 1 && lane <= L) {
    const float *col = lane < L ? lg + lane : lossb;  // lane L: the losses
    const int st = lane < L ? L : 1;
    float p8[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) p8[k] = 0.f;
    int b = 0;
    for (; b + 8 <= Bt; b += 8)
#pragma unroll
      for (int k = 0; k < 8; ++k) p8[k] += col[(b + k) * st];
#pragma unroll
    for (int k = 0; k < 8; ++k)
      if (b + k < Bt) p8[k] += col[(b + k) * st];
    const float sm = ((p8[0] + p8[1]) + (p8[2] + p8[3])) + ((p8[4] + p8[5]) + (p8[6] + p8[7]));
    if (lane < L) g[b_off + lane] = sm;
    else loss[rep] = sm / (float)Bt;
  }

  // input gradient of each example, weight-gradient share of each wave
  float acc[LM][4];
#pragma unroll
  for (int j = 0; j < LM; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[j][e] = 0.f;
  float *dhr = dh + (int64_t)rep * Bt * Ch + cl;
#pragma unroll
  for (int u = 0; u < NB; ++u) head_load4(hr + (int64_t)min(wave + u * NW, Bt - 1) * Ch, xn[u]);
  for (int b0 = wave; b0 < Bt; b0 += NB * NW) {
    float x[NB][4], d[NB][LM];
#pragma unroll
    for (int u = 0; u < NB; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) x[u][e] = xn[u][e];
#pragma unroll
    for (int u = 0; u < NB; ++u) head_load4(hr + (int64_t)min(b0 + (NB + u) * NW, Bt - 1) * Ch, xn[u]);
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      const int b = b0 + u * NW, bc = min(b, Bt - 1);
#pragma unroll
      for (int j = 0; j < LM; ++j) {
        const float v = lg[bc * L + min(j, L - 1)];
        d[u][j] = (b < Bt && j < L) ? v : 0.f;
      }
    }
    float o[NB][4];
#pragma unroll
    for (int u = 0; u < NB; ++u) {
#pragma unroll
      for (int e = 0; e < 4; ++e) o[u][e] = 0.f;
#pragma unroll
      for (int j = 0; j < LM; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          o[u][e] = fmaf(d[u][j], w[j][e], o[u][e]);
          acc[j][e] = fmaf(d[u][j], x[u][e], acc[j][e]);
        }
    }
    if (live) {
#pragma unroll
      for (int u = 0; u < NB; ++u)
        if (b0 + u * NW < Bt)
          *reinterpret_cast<float4 *>(dhr + (int64_t)(b0 + u * NW) * Ch) = make_float4(o[u][0], o[u][1], o[u][2], o[u][3]);
    }
  }
  // waves [half, 2 half) hand their sums to waves [0, half)
#pragma unroll
  for (int half = NW / 2; half >= 1; half >>= 1) {
    if (wave >= half && wave < 2 * half) {
#pragma unroll
      for (int j = 0; j < LM; ++j)
        if (j < L) red[((wave - half) * L + j) * 64 + lane] = make_float4(acc[j][0], acc[j][1], acc[j][2], acc[j][3]);
    }
    __syncthreads();
    if (wave < half) {
#pragma unroll
      for (int j = 0; j < LM; ++j) {
        const float4 r = red[(wave * L + min(j, L - 1)) * 64 + lane];
        acc[j][0] += r.x;
        acc[j][1] += r.y;
        acc[j][2] += r.z;
        acc[j][3] += r.w;
      }
    }
    __syncthreads();
  }
  if (wave == 0 && live) {
#pragma unroll
    for (int j = 0; j < LM; ++j)
      if (j < L)
#pragma unroll
        for (int e = 0; e < 4; ++e) g[w_off + (int64_t)j * Ch + c0 + e] = acc[j][e];
  }
}

template <typename T>
static hipError_t launch_linear_ce_reg(const T *h, const int32_t *y, const float *theta, int64_t P, int64_t w_off,
                                       int64_t b_off, float *grad, float *dh, float *loss, int C,
                                       const int32_t *rmap, int Bt, int Ch, int L, float eps, hipStream_t s) {
  const size_t shm = linear_ce_reg_lds_bytes(Bt, L);
  auto go = [&](auto kern) -> hipError_t {
    if (shm > 64 * 1024) {
      const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kern, dim3(C), dim3(kHeadRegWaves * 64), shm, s, h, y, theta, P, w_off, b_off, grad, dh,
                       loss, rmap, Bt, Ch, L, eps);
    return hipGetLastError();
  };
  switch ((L + 3) / 4) {
    case 1: return go(linear_ce_reg_kernel<T, 4>);
    case 2: return go(linear_ce_reg_kernel<T, 8>);
    case 3: return go(linear_ce_reg_kernel<T, 12>);
    default: return go(linear_ce_reg_kernel<T, 16>);
  }
}

// Gradient of the head pooling, with the last conv's ReLU mask:
// gpre = mask * route(dh / npos) (route = first maximum if max pooled).  A
// thread handles one 16-byte vector of channels of one window (max pooled)
// or one position.
// With routing codes (code, one byte per pooled element in the pooled
// layout: the window position of the first maximum, 4 for none) the head
// conv's output is not read.
template <typename T>
__global__ void __launch_bounds__(256)
head_pool_bwd_kernel(const T *__restrict__ a, const float *__restrict__ dh, T *__restrict__ gpre,
                     const int32_t *__restrict__ rmap, int64_t a_rs, int64_t dh_rs, uint32_t total, PoolIdx d, int W,
                     int Ch, int maxpool, const uint8_t *__restrict__ code, int64_t code_rs) {
  constexpr int VEC = ElemT<T>::VEC;
  const uint32_t i = blockIdx.x * 256u + threadIdx.x;
  if (i >= total) return;
  const int rep = replica_of(rmap, blockIdx.y);
  a += rep * a_rs;
  gpre += rep * a_rs;
  dh += rep * dh_rs;
  if (maxpool) {
    uint32_t bi;
    int cv;
    const int64_t base = pool_base(i, d, W, Ch, VEC, &bi, &cv);
    const float npos = (float)(d.ho.d * d.wo.d);
    const float *dr = dh + (int64_t)bi * Ch + cv * VEC;
    Vec16<T> g;
#pragma unroll
    for (int e = 0; e < VEC; ++e) g.v[e] = ElemT<T>::from_f(dr[e] / npos);
    if (code) {
      uint8_t k8[VEC];
      const uint8_t *cp = code + rep * code_rs + (int64_t)i * VEC;
      if constexpr (VEC == 8) {
        const uint2 cw = *reinterpret_cast<const uint2 *>(cp);
#pragma unroll
        for (int e = 0; e < 8; ++e) k8[e] = (uint8_t)(((e < 4 ? cw.x : cw.y) >> (8 * (e & 3))) & 0xffu);
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) k8[e] = cp[e];
      }
      const int64_t o[4] = {base, base + Ch, base + (int64_t)W * Ch, base + (int64_t)W * Ch + Ch};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        Vec16<T> out;
#pragma unroll
        for (int e = 0; e < VEC; ++e) out.v[e] = k8[e] == k ? g.v[e] : T(0);
        st16(gpre + o[k], out);
      }
    } else {
      route_window(a, gpre, base, W, Ch, g);
    }
  } else {
    // d.wo = W, d.ho = H: i = ((bi * H + h) * W + w) * CV + cv
    const uint32_t r = fdiv(i, d.cv);
    const int cv = (int)(i - r * d.cv.d);
    const uint32_t bi = fdiv(fdiv(r, d.wo), d.ho);
    const float npos = (float)(d.ho.d * d.wo.d);
    const float *dr = dh + (int64_t)bi * Ch + cv * VEC;
    const Vec16<T> v = ld16(a + (int64_t)i * VEC);
    Vec16<T> out;
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const T g = ElemT<T>::from_f(dr[e] / npos);
      out.v[e] = ElemT<T>::to_f(v.v[e]) > 0.f ? g : T(0);
    }
    st16(gpre + (int64_t)i * VEC, out);
  }
}

// ------------------------------------------------------------------- SGD
// g <- g + wd theta (weight decay); v <- mu v + g; theta <- theta - lr v, or
// theta - lr (g + mu v) with the Nesterov term (Sec. V-A), on the P
// parameters of the replica of slot blockIdx.y.  VEC divides P, so every
// replica row stays aligned.  The pass runs by segments of the parameter
// vector (sgd_seg_kernel) and also sums the split-K partials of the weight
// gradients: the ordered sum over the splits, from zero in split order, the
// partials of 8 splits loaded before they are added.
template <int VEC> struct FVec;
template <> struct FVec<1> { typedef float T; };
template <> struct FVec<2> { typedef float2 T; };
template <> struct FVec<4> { typedef float4 T; };

// one parameter's update
__device__ __forceinline__ void sgd_update(float &t, float &v, float g, float lr, float mu, float wd, int nesterov) {
  const float ge = g + wd * t;
  v = mu * v + ge;
  t -= lr * (nesterov ? ge + mu * v : v);
}

// SGD by segments (SgdSeg): the split-K partials of a weight gradient are
// summed here, in split order from zero (the partials of 8 splits loaded
// before they are added), and the sum is written to grad before the update.
// The block's segment is the last one whose first block is at most
// blockIdx.x.
template <int VEC>
__global__ void __launch_bounds__(256)
sgd_seg_kernel(float *__restrict__ theta, float *__restrict__ mom, float *__restrict__ grad,
               const float *__restrict__ part, const SgdSeg *__restrict__ segs, int nseg, int split_elems,
               int64_t P, const int32_t *__restrict__ rmap, float lr, float mu, float wd, int nesterov) {
  typedef typename FVec<VEC>::T V;
  int lo = 0, hi = nseg - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (segs[mid].first_block <= (int)blockIdx.x) lo = mid;
    else hi = mid - 1;
  }
  const SgdSeg sg = segs[lo];
  const int rep = replica_of(rmap, blockIdx.y);
  const int64_t base = (int64_t)rep * P + sg.begin;
  const int be = sg.splits > 0 ? split_elems : kSgdBlockElems;
  const int64_t e0 = ((int64_t)blockIdx.x - sg.first_block) * be;
  const int64_t e1 = min(sg.len, e0 + (int64_t)be);
  const float *pr = part + sg.src + (int64_t)rep * sg.rs;
  for (int64_t e = e0 + (int64_t)threadIdx.x * VEC; e < e1; e += 256 * VEC) {
    V g;
    if (sg.splits > 0) {
      float *gs = reinterpret_cast<float *>(&g);
#pragma unroll
      for (int q = 0; q < VEC; ++q) gs[q] = 0.f;
      int k = 0;
      for (; k + 8 <= sg.splits; k += 8) {
        V pv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) pv[u] = *reinterpret_cast<const V *>(pr + (k + u) * sg.ss + e);
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
          for (int q = 0; q < VEC; ++q) gs[q] += reinterpret_cast<const float *>(&pv[u])[q];
      }
      for (; k < sg.splits; ++k) {
        const V pv = *reinterpret_cast<const V *>(pr + k * sg.ss + e);
#pragma unroll
        for (int q = 0; q < VEC; ++q) gs[q] += reinterpret_cast<const float *>(&pv)[q];
      }
      *reinterpret_cast<V *>(grad + base + e) = g;
    } else {
      g = *reinterpret_cast<const V *>(grad + base + e);
    }
    V v = *reinterpret_cast<const V *>(mom + base + e), t = *reinterpret_cast<const V *>(theta + base + e);
    float *vf = reinterpret_cast<float *>(&v), *tf = reinterpret_cast<float *>(&t);
    const float *gf = reinterpret_cast<const float *>(&g);
#pragma unroll
    for (int q = 0; q < VEC; ++q) sgd_update(tf[q], vf[q], gf[q], lr, mu, wd, nesterov);
    *reinterpret_cast<V *>(mom + base + e) = v;
    *reinterpret_cast<V *>(theta + base + e) = t;
  }
}

// ---------------------------------------------------------------- fusion
// Eq. 5: theta_bar[p] = (sum_n w_n theta_n[p]) / W in fp64, in cluster order,
// rounded once to fp32 and written back to every replica.  A thread handles
// VEC consecutive parameters (VEC divides P, so every replica row stays
// aligned) and issues the loads of 16 replicas before it accumulates them.
// The weights come from device memory, or (KW, at most kMaxArgWeights
// replicas) from the kernel arguments.
struct FuseWeights {
  double w[kMaxArgWeights];
};

template <int VEC, bool KW>
__global__ void __launch_bounds__(256)
fuse_kernel(float *__restrict__ theta, const double *__restrict__ w, FuseWeights kw, double W, int C, int64_t P) {
  typedef typename FVec<VEC>::T V;
  constexpr int U = 16;
  const int64_t nv = P / VEC;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < nv;
       i += (int64_t)gridDim.x * blockDim.x) {
    double acc[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = 0.0;
    for (int n0 = 0; n0 < C; n0 += U) {
      V v[U];
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (n0 + u < C) v[u] = reinterpret_cast<const V *>(theta + (int64_t)(n0 + u) * P)[i];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (n0 + u < C) {
          const double wn = KW ? kw.w[n0 + u] : w[n0 + u];
          const float *f = reinterpret_cast<const float *>(&v[u]);
#pragma unroll
          for (int e = 0; e < VEC; ++e) acc[e] += wn * (double)f[e];
        }
      }
    }
    V out;
    float *o = reinterpret_cast<float *>(&out);
#pragma unroll
    for (int e = 0; e < VEC; ++e) o[e] = (float)(acc[e] / W);
    for (int n = 0; n < C; ++n) reinterpret_cast<V *>(theta + (int64_t)n * P)[i] = out;
  }
}

// The two halves of the same fusion, for a run whose replicas are spread
// over several devices: partial[p] = sum_n w_n theta_n[p] in fp64 in cluster
// order (the same operations as fuse_kernel), then theta_n[p] =
// fp32(partial[p] / W) for every replica.  A sharded run sums the devices'
// partials in between; on one device the two halves give fuse_kernel's
// result bit for bit.
template <int VEC, bool KW>
__global__ void __launch_bounds__(256)
fuse_partial_kernel(const float *__restrict__ theta, double *__restrict__ partial, const double *__restrict__ w,
                    FuseWeights kw, int C, int64_t P) {
  typedef typename FVec<VEC>::T V;
  constexpr int U = 16;
  const int64_t nv = P / VEC;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < nv;
       i += (int64_t)gridDim.x * blockDim.x) {
    double acc[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = 0.0;
    for (int n0 = 0; n0 < C; n0 += U) {
      V v[U];
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (n0 + u < C) v[u] = reinterpret_cast<const V *>(theta + (int64_t)(n0 + u) * P)[i];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (n0 + u < C) {
          const double wn = KW ? kw.w[n0 + u] : w[n0 + u];
          const float *f = reinterpret_cast<const float *>(&v[u]);
#pragma unroll
          for (int e = 0; e < VEC; ++e) acc[e] += wn * (double)f[e];
        }
      }
    }
#pragma unroll
    for (int e = 0; e < VEC; ++e) partial[i * VEC + e] = acc[e];
  }
}

template <int VEC>
__global__ void __launch_bounds__(256)
fuse_finalise_kernel(float *__restrict__ theta, const double *__restrict__ partial, double W, int C, int64_t P) {
  typedef typename FVec<VEC>::T V;
  const int64_t nv = P / VEC;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < nv;
       i += (int64_t)gridDim.x * blockDim.x) {
    V out;
    float *o = reinterpret_cast<float *>(&out);
#pragma unroll
    for (int e = 0; e < VEC; ++e) o[e] = (float)(partial[i * VEC + e] / W);
    for (int n = 0; n < C; ++n) reinterpret_cast<V *>(theta + (int64_t)n * P)[i] = out;
  }
}

inline unsigned grid_for(int64_t n, int per = 256, unsigned cap = 65535u * 8u) {
  const int64_t g = (n + per - 1) / per;
  return (unsigned)(g < 1 ? 1 : (g > cap ? cap : g));
}

}  // namespace

hipError_t launch_sample(const int32_t *ids, const int64_t *off, const int32_t *coe,
                         const int32_t *labels, const int64_t *ghist, int32_t *idx, int32_t *y, int32_t *hits,
                         int64_t *dev, int C, int B, int K, int L, int64_t nex, uint64_t seed, int64_t step0,
                         int nsteps, int64_t max_steps, int64_t R, hipStream_t s) {
  if (L < 1 || L > kMaxDevClasses || K > 32 * kMaxBitmapWords) return hipErrorInvalidValue;
  hipLaunchKernelGGL(sample_kernel, dim3(C, nsteps), dim3(256), 0, s, ids, off, coe, labels, ghist, idx, y,
                     hits, dev, C, B, K, L, nex, seed, step0, max_steps, R);
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
  const size_t padded = sizeof(float) * (size_t)(H + 2) * (W + 2) * Cin;
  const int n4 = (H * W * Cin) / 4, nv4 = (n4 + 255) / 256;
  if (Cin == 3 && padded <= 64 * 1024 && (H * W * Cin) % 4 == 0 && nv4 <= 4 && rows > 0) {
    // two examples per workgroup once that still leaves >= 4 workgroups per CU
    // (measured: 1 per workgroup 4.0 TB/s, 2: 4.5 TB/s, 4: 4.2 TB/s)
    const int per = rows >= 2048 ? 2 : 1;
    const dim3 grid((unsigned)((rows + per - 1) / per));
    const FastDiv fw = make_fastdiv((uint32_t)W);
#define GIM_GO(TT, KCC, NV)                                                                                    \
  hipLaunchKernelGGL((gather_im2col_fixed_kernel<TT, 3, KCC, NV>), grid, dim3(256), padded, s, images, idx,   \
                     (TT *)x, H, W, fw, rows, per)
#define GIM_NV(TT, KCC)                                                                                        \
  do {                                                                                                         \
    if (nv4 == 1) GIM_GO(TT, KCC, 1); else if (nv4 == 2) GIM_GO(TT, KCC, 2);                                   \
    else if (nv4 == 3) GIM_GO(TT, KCC, 3); else GIM_GO(TT, KCC, 4);                                            \
  } while (0)
    if (dtype == GCPSL_BF16 && Kc == 32) {
      GIM_NV(bf16_t, 32);
      return hipGetLastError();
    }
    if (dtype == GCPSL_F32 && Kc == 28) {
      GIM_NV(float, 28);
      return hipGetLastError();
    }
#undef GIM_NV
#undef GIM_GO
  }
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

void prep_add_layer(PrepJobs &jobs, int64_t w_off, int co, int ci, void *wf, int Kp, void *wd, int Kdp, int taps) {
  if (jobs.n + 2 > kMaxPrepJobs) return;  // the plan checks the layer count
  if (wd && co % 8 == 0 && ci % 8 == 0 && taps == 9) {
    // one read of the masters for both copies, 8-element (16-byte bf16) runs
    jobs.j[jobs.n++] = PrepJob{w_off, wd, co, ci, Kdp, 2, jobs.total, wf, Kp};
    jobs.total += ((co + 63) / 64) * ((ci + 63) / 64) * 9;
    return;
  }
  jobs.j[jobs.n++] = PrepJob{w_off, wf, co, ci, Kp, 0, jobs.total, nullptr, 0, taps};
  jobs.total += co;
  if (wd) {
    jobs.j[jobs.n++] = PrepJob{w_off, wd, co, ci, Kdp, 1, jobs.total, nullptr, 0, taps};
    jobs.total += ((co + 63) / 64) * ((ci + 63) / 64) * taps;
  }
}

hipError_t launch_prep_weights(int dtype, const float *theta, int64_t P, int C, const int32_t *rmap,
                               const PrepJobs &jobs, hipStream_t s) {
  if (jobs.n == 0) return hipSuccess;
  const dim3 grid((unsigned)jobs.total, C);
  if (dtype == GCPSL_BF16)
    hipLaunchKernelGGL(prep_weights_kernel<bf16_t>, grid, dim3(256), 0, s, theta, rmap, P, jobs);
  else
    hipLaunchKernelGGL(prep_weights_kernel<float>, grid, dim3(256), 0, s, theta, rmap, P, jobs);
  return hipGetLastError();
}

static PoolIdx pool_idx(int cv, int wo, int ho) { return PoolIdx{make_fastdiv(cv), make_fastdiv(wo), make_fastdiv(ho)}; }

// Elementwise pool kernels: grid (vectors of one replica / 256, replica
// slots).  A replica's tensors stay below 2 GiB, so its vector count fits
// 32 bits.
template <typename T>
static hipError_t maxpool_fwd_t(const T *x, T *z, int C, const int32_t *rmap, int Bt, int H, int W, int Ch,
                                hipStream_t s) {
  constexpr int VEC = ElemT<T>::VEC;
  const int Ho = H / 2, Wo = W / 2, CV = Ch / VEC;
  const uint32_t tot = (uint32_t)((int64_t)Bt * Ho * Wo * CV);
  hipLaunchKernelGGL(maxpool_fwd_kernel<T>, dim3((tot + 255) / 256, C), dim3(256), 0, s, x, z, rmap,
                     (int64_t)Bt * H * W * Ch, (int64_t)Bt * Ho * Wo * Ch, tot, pool_idx(CV, Wo, Ho), W, Ch);
  return hipGetLastError();
}

template <typename T>
static hipError_t maxpool_bwd_t(const T *a, const T *gz, T *gpre, int C, const int32_t *rmap, int Bt, int H, int W,
                                int Ch, hipStream_t s) {
  constexpr int VEC = ElemT<T>::VEC;
  const int Ho = H / 2, Wo = W / 2, CV = Ch / VEC;
  const uint32_t tot = (uint32_t)((int64_t)Bt * Ho * Wo * CV);
  hipLaunchKernelGGL(maxpool_bwd_kernel<T>, dim3((tot + 255) / 256, C), dim3(256), 0, s, a, gz, gpre, rmap,
                     (int64_t)Bt * H * W * Ch, (int64_t)Bt * Ho * Wo * Ch, tot, pool_idx(CV, Wo, Ho), W, Ch);
  return hipGetLastError();
}

template <typename T>
static hipError_t head_pool_t(const T *a, T *h, int C, const int32_t *rmap, int Bt, int H, int W, int Ch,
                              int maxpool, hipStream_t s) {
  constexpr int VEC = ElemT<T>::VEC;
  const int CV = Ch / VEC, CVB = std::min(CV, 256);
  hipLaunchKernelGGL(head_pool_kernel<T>, dim3((unsigned)Bt, (unsigned)((CV + CVB - 1) / CVB), (unsigned)C), dim3(256),
                     0, s, a, h, rmap, Bt, H, W, Ch, CVB, maxpool);
  return hipGetLastError();
}

template <typename T>
static hipError_t head_pool_bwd_t(const T *a, const float *dh, T *gpre, int C, const int32_t *rmap, int Bt, int H,
                                  int W, int Ch, int maxpool, hipStream_t s, const uint8_t *code, int64_t code_rs) {
  constexpr int VEC = ElemT<T>::VEC;
  const int CV = Ch / VEC;
  const int Ho = maxpool ? H / 2 : H, Wo = maxpool ? W / 2 : W;
  const uint32_t tot = (uint32_t)((int64_t)Bt * Ho * Wo * CV);
  if (code && (!maxpool || (reinterpret_cast<uintptr_t>(code) | (uintptr_t)code_rs) % VEC != 0))
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(head_pool_bwd_kernel<T>, dim3((tot + 255) / 256, C), dim3(256), 0, s, a, dh, gpre, rmap,
                     (int64_t)Bt * H * W * Ch, (int64_t)Bt * Ch, tot, pool_idx(CV, Wo, Ho), W, Ch, maxpool, code,
                     code_rs);
  return hipGetLastError();
}

hipError_t launch_maxpool_fwd(int dtype, const void *x, void *z, int C, const int32_t *rmap, int Bt, int H, int W,
                              int Ch, hipStream_t s) {
  if (dtype == GCPSL_BF16) return maxpool_fwd_t((const bf16_t *)x, (bf16_t *)z, C, rmap, Bt, H, W, Ch, s);
  return maxpool_fwd_t((const float *)x, (float *)z, C, rmap, Bt, H, W, Ch, s);
}

hipError_t launch_maxpool_bwd(int dtype, const void *a, const void *gz, void *gpre, int C, const int32_t *rmap,
                              int Bt, int H, int W, int Ch, hipStream_t s) {
  if (dtype == GCPSL_BF16)
    return maxpool_bwd_t((const bf16_t *)a, (const bf16_t *)gz, (bf16_t *)gpre, C, rmap, Bt, H, W, Ch, s);
  return maxpool_bwd_t((const float *)a, (const float *)gz, (float *)gpre, C, rmap, Bt, H, W, Ch, s);
}

hipError_t launch_head_pool(int dtype, const void *a, void *h, int C, const int32_t *rmap, int Bt, int H, int W,
                            int Ch, int maxpool, hipStream_t s) {
  if (dtype == GCPSL_BF16) return head_pool_t((const bf16_t *)a, (bf16_t *)h, C, rmap, Bt, H, W, Ch, maxpool, s);
  return head_pool_t((const float *)a, (float *)h, C, rmap, Bt, H, W, Ch, maxpool, s);
}

hipError_t launch_linear_ce(int dtype, const void *h, const int32_t *y, const float *theta, int64_t P,
                            int64_t w_off, int64_t b_off, float *grad, float *dh, float *loss, int C,
                            const int32_t *rmap, int Bt, int Ch, int L, float eps, hipStream_t s) {
  if (linear_ce_reg_ok(Bt, Ch, L))
    return dtype == GCPSL_BF16 ? launch_linear_ce_reg((const bf16_t *)h, y, theta, P, w_off, b_off, grad, dh, loss,
                                                      C, rmap, Bt, Ch, L, eps, s)
                               : launch_linear_ce_reg((const float *)h, y, theta, P, w_off, b_off, grad, dh, loss,
                                                      C, rmap, Bt, Ch, L, eps, s);
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
                       theta, P, w_off, b_off, grad, dh, loss, rmap, Bt, Ch, L, eps);
  else
    hipLaunchKernelGGL(linear_ce_kernel<float>, dim3(C), dim3(1024), shm, s, (const float *)h, y,
                       theta, P, w_off, b_off, grad, dh, loss, rmap, Bt, Ch, L, eps);
  return hipGetLastError();
}

hipError_t launch_head_pool_bwd(int dtype, const void *a, const float *dh, void *gpre, int C, const int32_t *rmap,
                                int Bt, int H, int W, int Ch, int maxpool, hipStream_t s, const uint8_t *code,
                                int64_t code_rs) {
  if (dtype == GCPSL_BF16)
    return head_pool_bwd_t((const bf16_t *)a, dh, (bf16_t *)gpre, C, rmap, Bt, H, W, Ch, maxpool, s, code, code_rs);
  return head_pool_bwd_t((const float *)a, dh, (float *)gpre, C, rmap, Bt, H, W, Ch, maxpool, s, code, code_rs);
}

hipError_t launch_sgd_seg(float *theta, float *mom, float *grad, const float *partials, const SgdSeg *segs, int nseg,
                          int blocks, int vec, int split_elems, int64_t P, int C, const int32_t *rmap, float lr,
                          float mu, float wd, int nesterov, hipStream_t s) {
  if (nseg < 1 || blocks < 1 || split_elems < 1) return hipErrorInvalidValue;
  // vec (4, 2 or 1) divides P and every segment's start, length, partial
  // offset and strides (the plan's choice); the pointers must allow it too
  const uintptr_t al = reinterpret_cast<uintptr_t>(theta) | reinterpret_cast<uintptr_t>(mom) |
                       reinterpret_cast<uintptr_t>(grad) | reinterpret_cast<uintptr_t>(partials);
  if (vec == 4 && al % 16 != 0) vec = al % 8 == 0 ? 2 : 1;
  if (vec == 2 && al % 8 != 0) vec = 1;
  const dim3 g((uint32_t)blocks, (uint32_t)C);
  if (vec == 4)
    hipLaunchKernelGGL(sgd_seg_kernel<4>, g, dim3(256), 0, s, theta, mom, grad, partials, segs, nseg, split_elems, P,
                       rmap, lr, mu, wd, nesterov);
  else if (vec == 2)
    hipLaunchKernelGGL(sgd_seg_kernel<2>, g, dim3(256), 0, s, theta, mom, grad, partials, segs, nseg, split_elems, P,
                       rmap, lr, mu, wd, nesterov);
  else
    hipLaunchKernelGGL(sgd_seg_kernel<1>, g, dim3(256), 0, s, theta, mom, grad, partials, segs, nseg, split_elems, P,
                       rmap, lr, mu, wd, nesterov);
  return hipGetLastError();
}

// One thread per VEC parameters up to 65536 workgroups (a fully resident
// grid streams ~2 % faster than 16384 workgroups looping over the rows).
hipError_t launch_fuse_partial(const float *theta, double *partial, const double *w_dev, const double *w_host,
                               int C, int64_t P, hipStream_t s) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(theta);
  FuseWeights kw{};
  const bool by_arg = w_host && C <= kMaxArgWeights;
  if (by_arg)
    for (int n = 0; n < C; ++n) kw.w[n] = w_host[n];
  else if (!w_dev)
    return hipErrorInvalidValue;
#define FUSE_GO(VEC)                                                                                        \
  do {                                                                                                      \
    const dim3 g(grid_for(P / VEC, 256, 65536));                                                           \
    if (by_arg)                                                                                             \
      hipLaunchKernelGGL((fuse_partial_kernel<VEC, true>), g, dim3(256), 0, s, theta, partial, w_dev, kw, C, P); \
    else                                                                                                    \
      hipLaunchKernelGGL((fuse_partial_kernel<VEC, false>), g, dim3(256), 0, s, theta, partial, w_dev, kw, C, P); \
  } while (0)
  if (P % 4 == 0 && a % 16 == 0)
    FUSE_GO(4);
  else if (P % 2 == 0 && a % 8 == 0)
    FUSE_GO(2);
  else
    FUSE_GO(1);
#undef FUSE_GO
  return hipGetLastError();
}

hipError_t launch_fuse_finalise(float *theta, const double *partial, double W, int C, int64_t P, hipStream_t s) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(theta);
#define FUSE_GO(VEC)                                                                                     \
  hipLaunchKernelGGL((fuse_finalise_kernel<VEC>), dim3(grid_for(P / VEC, 256, 65536)), dim3(256), 0, s, \
                     theta, partial, W, C, P)
  if (P % 4 == 0 && a % 16 == 0)
    FUSE_GO(4);
  else if (P % 2 == 0 && a % 8 == 0)
    FUSE_GO(2);
  else
    FUSE_GO(1);
#undef FUSE_GO
  return hipGetLastError();
}

hipError_t launch_fuse(float *theta, const double *w_dev, const double *w_host, double W, int C, int64_t P,
                       hipStream_t s) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(theta);
  FuseWeights kw{};
  const bool by_arg = w_host && C <= kMaxArgWeights;
  if (by_arg)
    for (int n = 0; n < C; ++n) kw.w[n] = w_host[n];
  else if (!w_dev)
    return hipErrorInvalidValue;
#define FUSE_GO(VEC)                                                                                     \
  do {                                                                                                   \
    const dim3 g(grid_for(P / VEC, 256, 65536));                                                        \
    if (by_arg) hipLaunchKernelGGL((fuse_kernel<VEC, true>), g, dim3(256), 0, s, theta, w_dev, kw, W, C, P); \
    else hipLaunchKernelGGL((fuse_kernel<VEC, false>), g, dim3(256), 0, s, theta, w_dev, kw, W, C, P);      \
  } while (0)
  if (P % 4 == 0 && a % 16 == 0)
    FUSE_GO(4);
  else if (P % 2 == 0 && a % 8 == 0)
    FUSE_GO(2);
  else
    FUSE_GO(1);
#undef FUSE_GO
  return hipGetLastError();
}
