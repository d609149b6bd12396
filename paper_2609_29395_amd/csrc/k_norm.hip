// Normalisation layers of the split CNN (Sec. IV-B): GroupNorm in the client
// segment, BatchNorm in the server segment, each followed by ReLU, over the
// raw output z [Bt][H][W][Ch] (NHWC) of the conv before it:
//
//   x_hat = (z - mean) * rstd,  rstd = 1 / sqrt(var + 1e-5),  var biased,
//   u = gamma_c x_hat + beta_c,  a = ReLU(u);
//
// batch norm takes mean and var per channel over (Bt, H, W), group norm per
// example over (H, W, the channels of a group).  Backward, from du = dL/du:
//
//   dgamma_c = sum du x_hat,  dbeta_c = sum du        (over Bt, H, W)
//   dz = rstd (du gamma_c - S1 / n - x_hat S2 / n),
//   S1 = sum du gamma_c,  S2 = sum du gamma_c x_hat   (over the set of n values)
//
// Batch norm also updates its replica's running statistics (momentum 0.1,
// unbiased variance for the running value) and batch counter.
//
// Every sum runs in fp64 in a fixed order (per-thread pixel strides, then
// pixel-lane order within a workgroup; across the chunks of a channel
// reduction, eight strided chunk lanes, then lane order), so results do not
// depend on scheduling or on which replicas share a launch.  A thread owns
// one 16-byte vector of VEC channels; a workgroup has 256 / (Ch / VEC) pixel
// lanes.  Chunks shrink for small tensors (16 to 256 pixels) so that late,
// low-resolution layers still spread over the chip.
#include "runtime.h"

namespace {

constexpr double kEps = 1e-5;
constexpr double kMomentum = 0.1;

template <typename T> struct V16 {
  T v[ElemT<T>::VEC];
};
template <typename T> __device__ __forceinline__ V16<T> load16(const T *p) {
  return __builtin_bit_cast(V16<T>, *reinterpret_cast<const uint4 *>(p));
}
template <typename T> __device__ __forceinline__ void store16(T *p, const V16<T> &v) {
  *reinterpret_cast<uint4 *>(p) = __builtin_bit_cast(uint4, v);
}

// statistics index of channel c of example b
__device__ __forceinline__ int stat_index(const NormArgs &a, int b, int c) {
  return a.groups ? b * a.groups + c / (a.Ch / a.groups) : c;
}

// Per-channel sums over one chunk of pixels: MODE 0 sum z and z^2 (batch
// statistics), MODE 1 sum du and du x_hat (gradients of gamma and beta).
// Partials part[rep][chunk][c][2].
template <typename T, int MODE>
__global__ void __launch_bounds__(256)
chan_reduce_kernel(NormArgs a, FastDiv fhw) {
  constexpr int VEC = ElemT<T>::VEC;
  __shared__ double red[256][2 * VEC];
  const int rep = replica_of(a.rmap, blockIdx.y);
  const int CV = a.Ch / VEC, PL = 256 / CV;
  const int tid = threadIdx.x, cv = tid % CV, pl = tid / CV;
  const int64_t M = (int64_t)a.Bt * a.H * a.W;
  const int64_t p0 = (int64_t)blockIdx.x * a.chunk_px, p1 = min(M, p0 + a.chunk_px);
  const T *z = reinterpret_cast<const T *>(a.z) + rep * a.z_rs;
  const T *du = reinterpret_cast<const T *>(a.du) + rep * a.z_rs;
  const float *mean = a.mean + (int64_t)rep * a.nstat, *rstd = a.rstd + (int64_t)rep * a.nstat;
  double s0[VEC], s1[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) s0[e] = s1[e] = 0.0;
  // MODE 1: the statistics of this thread's channels, loaded when its example
  // changes (group norm) or once (batch norm)
  int kb = -1;
  float km[VEC], kr[VEC];
  auto add = [&](const V16<T> &zv, const V16<T> &gv, int64_t p) {
    if constexpr (MODE == 0) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const double v = ElemT<T>::to_f(zv.v[e]);
        s0[e] += v;
        s1[e] += v * v;
      }
    } else {
      const int b = (int)fdiv((uint32_t)p, fhw);
      if (kb < 0 || (a.groups && b != kb)) {
        kb = b;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const int si = stat_index(a, b, cv * VEC + e);
          km[e] = mean[si], kr[e] = rstd[si];
        }
      }
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const float xh = (ElemT<T>::to_f(zv.v[e]) - km[e]) * kr[e];
        const double g = ElemT<T>::to_f(gv.v[e]);
        s0[e] += g;
        s1[e] += g * (double)xh;
      }
    }
  };
  if (pl < PL) {
    // four pixels' loads in flight, added in pixel order
    int64_t p = p0 + pl;
    for (; p + 3 * PL < p1; p += 4 * PL) {
      V16<T> zv[4], gv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        zv[u] = load16(z + (p + u * PL) * a.Ch + cv * VEC);
        if constexpr (MODE == 1) gv[u] = load16(du + (p + u * PL) * a.Ch + cv * VEC);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) add(zv[u], gv[u], p + u * PL);
    }
    for (; p < p1; p += PL) {
      V16<T> zv = load16(z + p * a.Ch + cv * VEC), gv{};
      if constexpr (MODE == 1) gv = load16(du + p * a.Ch + cv * VEC);
      add(zv, gv, p);
    }
  }
#pragma unroll
  for (int e = 0; e < VEC; ++e) {
    red[tid][e] = s0[e];
    red[tid][VEC + e] = s1[e];
  }
  __syncthreads();
  // the chunk's sums: one (channel, sum) per thread, over the pixel lanes in
  // lane order
  double *out = a.part + ((int64_t)rep * a.chunks + blockIdx.x) * a.Ch * 2;
  for (int o = tid; o < 2 * a.Ch; o += 256) {
    const int c = o >> 1, k = o & 1, ocv = c / VEC, e = c - ocv * VEC;
    double t = 0.0;
    for (int l = 0; l < PL; ++l) t += red[l * CV + ocv][k * VEC + e];
    out[o] = t;
  }
}

// Chunk partials -> per-channel sums.  A workgroup takes 32 channels: lane j
// of a channel adds chunks j, j + 8, j + 16, ... in order (four loads in
// flight), and the 8 lanes' sums are added in lane order.  MODE 0:
// batch-norm mean and rstd, and the running statistics; MODE 1: dbeta,
// dgamma into grad and (batch norm) the sums for the input gradient.
constexpr int kFinishCh = 32, kFinishLanes = 8;

template <int MODE>
__global__ void __launch_bounds__(256)
chan_finish_kernel(NormArgs a) {
  __shared__ double red[kFinishLanes][kFinishCh][2];
  const int rep = replica_of(a.rmap, blockIdx.y);
  const int cl = threadIdx.x % kFinishCh, j = threadIdx.x / kFinishCh;
  const int c = blockIdx.x * kFinishCh + cl;
  double S0 = 0.0, S1 = 0.0;
  if (c < a.Ch) {
    const double *pp = a.part + ((int64_t)rep * a.chunks * a.Ch + c) * 2;
    const int64_t step = (int64_t)a.Ch * 2;
    int k = j;
    for (; k + 3 * kFinishLanes < a.chunks; k += 4 * kFinishLanes) {
      double v[4][2];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        v[u][0] = pp[(k + u * kFinishLanes) * step];
        v[u][1] = pp[(k + u * kFinishLanes) * step + 1];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        S0 += v[u][0];
        S1 += v[u][1];
      }
    }
    for (; k < a.chunks; k += kFinishLanes) {
      S0 += pp[k * step];
      S1 += pp[k * step + 1];
    }
  }
  red[j][cl][0] = S0;
  red[j][cl][1] = S1;
  __syncthreads();
  if (j != 0 || c >= a.Ch) return;
  S0 = red[0][cl][0];
  S1 = red[0][cl][1];
#pragma unroll
  for (int l = 1; l < kFinishLanes; ++l) {
    S0 += red[l][cl][0];
    S1 += red[l][cl][1];
  }
  const double n = (double)a.Bt * a.H * a.W;
  if constexpr (MODE == 0) {
    const double mean = S0 / n;
    const double var = fmax(S1 / n - mean * mean, 0.0);
    a.mean[(int64_t)rep * a.nstat + c] = (float)mean;
    a.rstd[(int64_t)rep * a.nstat + c] = (float)(1.0 / sqrt(var + kEps));
    float *st = a.state + rep * a.S + a.st_off;
    st[c] = (float)((1.0 - kMomentum) * (double)st[c] + kMomentum * mean);
    st[a.Ch + c] = (float)((1.0 - kMomentum) * (double)st[a.Ch + c] + kMomentum * var * n / (n - 1.0));
    if (c == 0) st[2 * a.Ch] = (float)((double)st[2 * a.Ch] + 1.0);
  } else {
    a.grad[rep * a.P + a.b_off + c] = (float)S0;
    a.grad[rep * a.P + a.g_off + c] = (float)S1;
    if (!a.groups) {
      a.sums[((int64_t)rep * a.nstat + c) * 2] = S0;
      a.sums[((int64_t)rep * a.nstat + c) * 2 + 1] = S1;
    }
  }
}

// Group norm, one workgroup per example: MODE 0 mean and rstd per group;
// MODE 1 the sums S1 = sum du gamma, S2 = sum du gamma x_hat per group.
template <typename T, int MODE>
__global__ void __launch_bounds__(256)
group_reduce_kernel(NormArgs a) {
  constexpr int VEC = ElemT<T>::VEC;
  __shared__ double red[256][2 * VEC];
  __shared__ double chs[2048][2];  // per-channel sums (Ch <= 2048)
  const int rep = replica_of(a.rmap, blockIdx.y);
  const int b = blockIdx.x;
  const int CV = a.Ch / VEC, PL = 256 / CV;
  const int tid = threadIdx.x, cv = tid % CV, pl = tid / CV;
  const int HW = a.H * a.W, G = a.groups, CG = a.Ch / G;
  const int64_t base = rep * a.z_rs + (int64_t)b * HW * a.Ch;
  const T *z = reinterpret_cast<const T *>(a.z) + base;
  const T *du = reinterpret_cast<const T *>(a.du) + base;
  const float *mean = a.mean + (int64_t)rep * a.nstat, *rstd = a.rstd + (int64_t)rep * a.nstat;
  const float *gamma = a.theta + rep * a.P + a.g_off;
  double s0[VEC], s1[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) s0[e] = s1[e] = 0.0;
  // MODE 1: this thread's channels' statistics of example b and gamma
  float km[VEC], kr[VEC], kg[VEC];
  if constexpr (MODE == 1) {
    if (pl < PL) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const int c = cv * VEC + e, si = b * G + c / CG;
        km[e] = mean[si], kr[e] = rstd[si], kg[e] = gamma[c];
      }
    }
  }
  auto add = [&](const V16<T> &zv, const V16<T> &gv) {
    if constexpr (MODE == 0) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const double v = ElemT<T>::to_f(zv.v[e]);
        s0[e] += v;
        s1[e] += v * v;
      }
    } else {
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const float xh = (ElemT<T>::to_f(zv.v[e]) - km[e]) * kr[e];
        const double dx = (double)ElemT<T>::to_f(gv.v[e]) * kg[e];
        s0[e] += dx;
        s1[e] += dx * (double)xh;
      }
    }
  };
  if (pl < PL) {
    // four pixels' loads in flight, added in pixel order
    int p = pl;
    for (; p + 3 * PL < HW; p += 4 * PL) {
      V16<T> zv[4], gv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        zv[u] = load16(z + (int64_t)(p + u * PL) * a.Ch + cv * VEC);
        if constexpr (MODE == 1) gv[u] = load16(du + (int64_t)(p + u * PL) * a.Ch + cv * VEC);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) add(zv[u], gv[u]);
    }
    for (; p < HW; p += PL) {
      V16<T> zv = load16(z + (int64_t)p * a.Ch + cv * VEC), gv{};
      if constexpr (MODE == 1) gv = load16(du + (int64_t)p * a.Ch + cv * VEC);
      add(zv, gv);
    }
  }
#pragma unroll
  for (int e = 0; e < VEC; ++e) {
    red[tid][e] = s0[e];
    red[tid][VEC + e] = s1[e];
  }
  __syncthreads();
  // per-channel sums: one (channel, sum) per thread, over the pixel lanes in
  // lane order
  for (int o = tid; o < 2 * a.Ch; o += 256) {
    const int c = o >> 1, k = o & 1, ocv = c / VEC, e = c - ocv * VEC;
    double t = 0.0;
    for (int l = 0; l < PL; ++l) t += red[l * CV + ocv][k * VEC + e];
    chs[c][k] = t;
  }
  __syncthreads();
  for (int g = tid; g < G; g += blockDim.x) {
    double S0 = 0.0, S1 = 0.0;
    for (int c = g * CG; c < (g + 1) * CG; ++c) {
      S0 += chs[c][0];
      S1 += chs[c][1];
    }
    const int64_t si = (int64_t)rep * a.nstat + b * G + g;
    if constexpr (MODE == 0) {
      const double n = (double)HW * CG;
      const double m = S0 / n;
      const double var = fmax(S1 / n - m * m, 0.0);
      a.mean[si] = (float)m;
      a.rstd[si] = (float)(1.0 / sqrt(var + kEps));
    } else {
      a.sums[si * 2] = S0;
      a.sums[si * 2 + 1] = S1;
    }
  }
}

// The elementwise passes: a workgroup takes kApplyUnroll consecutive runs of
// 256 16-byte vectors (four loads in flight per thread), so a thread keeps
// the same VEC channels (256 is a multiple of the vectors per pixel) and
// stays within one example over neighbouring pixels.  The per-channel values
// it needs (gamma, beta; the statistics of its example for group norm) are
// loaded when its channels or its example change, not per element; every
// value and expression is the same as per element, so the results are too.
constexpr int kApplyUnroll = 4;

// a = ReLU(gamma (z - mean) rstd + beta (+ res)) (without the ReLU for a
// shortcut's norm).
template <typename T>
__global__ void __launch_bounds__(256)
norm_apply_fwd_kernel(NormArgs a, uint32_t total, FastDiv fcv, FastDiv fhw) {
  constexpr int VEC = ElemT<T>::VEC;
  const int rep = replica_of(a.rmap, blockIdx.y);
  const int CV = a.Ch / VEC;
  const T *z = reinterpret_cast<const T *>(a.z) + rep * a.z_rs;
  const T *res = a.res ? reinterpret_cast<const T *>(a.res) + rep * a.z_rs : nullptr;
  T *out = reinterpret_cast<T *>(a.a) + rep * a.z_rs;
  const float *mean = a.mean + (int64_t)rep * a.nstat, *rstd = a.rstd + (int64_t)rep * a.nstat;
  const float *gamma = a.theta + rep * a.P + a.g_off, *beta = a.theta + rep * a.P + a.b_off;
  constexpr uint32_t stride = 256u;
  int kc = -1, kb = -1;  // channel vector and example of the cached values
  float km[VEC], kr[VEC], kg[VEC], kbt[VEC];
  {
    const uint32_t i0 = blockIdx.x * (256u * kApplyUnroll) + threadIdx.x;
    V16<T> zv[kApplyUnroll], rv[kApplyUnroll];
#pragma unroll
    for (int u = 0; u < kApplyUnroll; ++u) {
      const uint32_t i = i0 + u * stride;
      if (i < total) {
        zv[u] = load16(z + (int64_t)i * VEC);
        if (res) rv[u] = load16(res + (int64_t)i * VEC);
      }
    }
#pragma unroll
    for (int u = 0; u < kApplyUnroll; ++u) {
      const uint32_t i = i0 + u * stride;
      if (i >= total) break;
      const uint32_t p = fdiv(i, fcv);  // pixel, then its example
      const int cv = (int)(i - p * CV), b = (int)fdiv(p, fhw);
      if (cv != kc || (a.groups && b != kb)) {
        kc = cv, kb = b;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const int c = cv * VEC + e, si = stat_index(a, b, c);
          km[e] = mean[si], kr[e] = rstd[si], kg[e] = gamma[c], kbt[e] = beta[c];
        }
      }
      V16<T> o;
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        float uu = kg[e] * ((ElemT<T>::to_f(zv[u].v[e]) - km[e]) * kr[e]) + kbt[e];
        if (res) uu += ElemT<T>::to_f(rv[u].v[e]);
        o.v[e] = ElemT<T>::from_f(a.relu ? fmaxf(uu, 0.f) : uu);
      }
      store16(out + (int64_t)i * VEC, o);
    }
  }
}

// dz = rstd (du gamma - S1 / n - x_hat S2 / n); batch norm's S1, S2 are gamma
// times the per-channel sums.
template <typename T>
__global__ void __launch_bounds__(256)
norm_apply_bwd_kernel(NormArgs a, uint32_t total, FastDiv fcv, FastDiv fhw) {
  constexpr int VEC = ElemT<T>::VEC;
  const int rep = replica_of(a.rmap, blockIdx.y);
  const int CV = a.Ch / VEC;
  const T *z = reinterpret_cast<const T *>(a.z) + rep * a.z_rs;
  const T *du = reinterpret_cast<const T *>(a.du) + rep * a.z_rs;
  T *dz = reinterpret_cast<T *>(a.dz) + rep * a.z_rs;
  const float *mean = a.mean + (int64_t)rep * a.nstat, *rstd = a.rstd + (int64_t)rep * a.nstat;
  const float *gamma = a.theta + rep * a.P + a.g_off;
  const double *sums = a.sums + (int64_t)rep * a.nstat * 2;
  const double n = a.groups ? (double)a.H * a.W * (a.Ch / a.groups) : (double)a.Bt * a.H * a.W;
  constexpr uint32_t stride = 256u;
  int kc = -1, kb = -1;
  float km[VEC], kr[VEC], kg[VEC], k1[VEC], k2[VEC];
  {
    const uint32_t i0 = blockIdx.x * (256u * kApplyUnroll) + threadIdx.x;
    V16<T> zv[kApplyUnroll], gv[kApplyUnroll];
#pragma unroll
    for (int u = 0; u < kApplyUnroll; ++u) {
      const uint32_t i = i0 + u * stride;
      if (i < total) {
        zv[u] = load16(z + (int64_t)i * VEC);
        gv[u] = load16(du + (int64_t)i * VEC);
      }
    }
#pragma unroll
    for (int u = 0; u < kApplyUnroll; ++u) {
      const uint32_t i = i0 + u * stride;
      if (i >= total) break;
      const uint32_t p = fdiv(i, fcv);  // pixel, then its example
      const int cv = (int)(i - p * CV), b = (int)fdiv(p, fhw);
      if (cv != kc || (a.groups && b != kb)) {
        kc = cv, kb = b;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const int c = cv * VEC + e, si = stat_index(a, b, c);
          km[e] = mean[si], kr[e] = rstd[si], kg[e] = gamma[c];
          k1[e] = (float)(sums[2 * si] / n), k2[e] = (float)(sums[2 * si + 1] / n);
        }
      }
      V16<T> o;
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const float xh = (ElemT<T>::to_f(zv[u].v[e]) - km[e]) * kr[e];
        const float v = a.groups ? kr[e] * (ElemT<T>::to_f(gv[u].v[e]) * kg[e] - k1[e] - xh * k2[e])
                                 : kr[e] * kg[e] * (ElemT<T>::to_f(gv[u].v[e]) - k1[e] - xh * k2[e]);
        o.v[e] = ElemT<T>::from_f(v);
      }
      store16(dz + (int64_t)i * VEC, o);
    }
  }
}

// workgroups of an elementwise pass over `total` vectors of one replica:
// about kApplyUnroll vectors per thread
uint32_t apply_blocks(uint32_t total) {
  return std::max<uint32_t>(1u, (total + 256u * kApplyUnroll - 1) / (256u * kApplyUnroll));
}

template <typename T>
hipError_t norm_fwd_t(const NormArgs &a, hipStream_t s) {
  constexpr int VEC = ElemT<T>::VEC;
  const uint32_t total = (uint32_t)((int64_t)a.Bt * a.H * a.W * (a.Ch / VEC));
  const FastDiv fcv = make_fastdiv((uint32_t)(a.Ch / VEC)), fhw = make_fastdiv((uint32_t)(a.H * a.W));
  if (a.groups) {
    hipLaunchKernelGGL((group_reduce_kernel<T, 0>), dim3(a.Bt, a.C), dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL((chan_reduce_kernel<T, 0>), dim3(a.chunks, a.C), dim3(256), 0, s, a, fhw);
    hipLaunchKernelGGL((chan_finish_kernel<0>), dim3((a.Ch + kFinishCh - 1) / kFinishCh, a.C), dim3(256), 0, s, a);
  }
  hipLaunchKernelGGL((norm_apply_fwd_kernel<T>), dim3(apply_blocks(total), a.C), dim3(256), 0, s, a, total, fcv, fhw);
  return hipGetLastError();
}

template <typename T>
hipError_t norm_bwd_t(const NormArgs &a, hipStream_t s) {
  constexpr int VEC = ElemT<T>::VEC;
  const uint32_t total = (uint32_t)((int64_t)a.Bt * a.H * a.W * (a.Ch / VEC));
  const FastDiv fcv = make_fastdiv((uint32_t)(a.Ch / VEC)), fhw = make_fastdiv((uint32_t)(a.H * a.W));
  hipLaunchKernelGGL((chan_reduce_kernel<T, 1>), dim3(a.chunks, a.C), dim3(256), 0, s, a, fhw);
  hipLaunchKernelGGL((chan_finish_kernel<1>), dim3((a.Ch + kFinishCh - 1) / kFinishCh, a.C), dim3(256), 0, s, a);
  if (a.groups) hipLaunchKernelGGL((group_reduce_kernel<T, 1>), dim3(a.Bt, a.C), dim3(256), 0, s, a);
  hipLaunchKernelGGL((norm_apply_bwd_kernel<T>), dim3(apply_blocks(total), a.C), dim3(256), 0, s, a, total, fcv, fhw);
  return hipGetLastError();
}

}  // namespace

bool norm_ok(int dtype, int Ch, int groups) {
  const int vec = dtype == GCPSL_BF16 ? 8 : 4;
  return Ch % vec == 0 && Ch / vec <= 256 && Ch <= 2048 && (groups == 0 || Ch % groups == 0);
}

hipError_t launch_norm_fwd(int dtype, const NormArgs &a, hipStream_t s) {
  return dtype == GCPSL_BF16 ? norm_fwd_t<bf16_t>(a, s) : norm_fwd_t<float>(a, s);
}

hipError_t launch_norm_bwd(int dtype, const NormArgs &a, hipStream_t s) {
  return dtype == GCPSL_BF16 ? norm_bwd_t<bf16_t>(a, s) : norm_bwd_t<float>(a, s);
}
