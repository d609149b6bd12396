// Replica-batched implicit-GEMM 3x3 convolutions on MFMA (gfx950).
//
// Every pass of a conv layer is a dense contraction:
//   forward  out[m][co] = sum_{(r,s,ci)} x[m + (r-1, s-1)][ci] W[co][r][s][ci]
//   dgrad    dx[m][ci]  = sum_{(r,s,co)} g[m + (r-1, s-1)][co] W[co][2-r][2-s][ci]
//            (a forward conv of g with the flipped, transposed weights)
//   wgrad    dW[co][(r,s,ci)] = sum_m g[m][co] x[m + (r-1, s-1)][ci]
// with m = (b, h, w) over the batch and the image.  One workgroup computes a
// BM x BN output tile of one replica; replicas are folded into the linear
// workgroup index, so one launch covers all C clusters.
//
// Tiles are staged through LDS in "k-contiguous" rows of 128 bytes (64 bf16
// or 32 fp32 k values) plus 16 bytes of padding, double buffered with one
// barrier per k tile.  4 waves in a 2x2 layout each own a (BM/2) x (BN/2)
// sub-tile of 16x16 MFMA blocks.  A lane's operand fragment is 8 consecutive
// k values of one row: one v_mfma_f32_16x16x32_bf16, or eight
// v_mfma_f32_16x16x4_f32 (lane group g feeds k = 8g + j to the j-th), so the
// fp32 and bf16 paths share the LDS layout and the tile loop.
#include "runtime.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

template <typename T> struct Frag;
template <> struct Frag<bf16_t> { uint4 q; };
template <> struct Frag<float> { float v[8]; };

__device__ __forceinline__ void load_frag(Frag<bf16_t> &f, const bf16_t *p) {
  f.q = *reinterpret_cast<const uint4 *>(p);
}
__device__ __forceinline__ void load_frag(Frag<float> &f, const float *p) {
  const uint4 x = *reinterpret_cast<const uint4 *>(p);
  const uint4 y = *reinterpret_cast<const uint4 *>(p + 4);
  f.v[0] = __uint_as_float(x.x); f.v[1] = __uint_as_float(x.y);
  f.v[2] = __uint_as_float(x.z); f.v[3] = __uint_as_float(x.w);
  f.v[4] = __uint_as_float(y.x); f.v[5] = __uint_as_float(y.y);
  f.v[6] = __uint_as_float(y.z); f.v[7] = __uint_as_float(y.w);
}

__device__ __forceinline__ void mma(f32x4_t &acc, const Frag<bf16_t> &a, const Frag<bf16_t> &b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a.q),
                                                __builtin_bit_cast(bf16x8_t, b.q), acc, 0, 0, 0);
}
__device__ __forceinline__ void mma(f32x4_t &acc, const Frag<float> &a, const Frag<float> &b) {
#pragma unroll
  for (int j = 0; j < 8; ++j) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[j], b.v[j], acc, 0, 0, 0);
}

template <typename T> struct Pack {
  T v[16 / sizeof(T)];
};

// Raw buffer access: an offset at or beyond the descriptor's byte count reads
// zero without touching memory.  Invalid lanes use kOob (tensors here are
// far below 2 GiB), so zero padding and ragged tiles need no branches.
constexpr uint32_t kOob = 0x80000000u;
constexpr int kBufferFlags = 0x00020000;  // raw 32-bit data format

// The descriptor must live in scalar registers; base and size are uniform
// across the workgroup, readfirstlane makes that explicit to the compiler.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
  const uint64_t p = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)p);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(p >> 32));
  void *q = reinterpret_cast<void *>(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(q, (short)0, (int)__builtin_amdgcn_readfirstlane(bytes), kBufferFlags);
}

__device__ __forceinline__ uint4 buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

// Shared tile geometry and the MFMA loop over one staged k tile.
template <typename T, int BM, int BN, int WM = 2, int WN = 2, int BKB = 128> struct Tile {
  static constexpr int VEC = ElemT<T>::VEC;
  static constexpr int BK = BKB / (int)sizeof(T);  // k values per staged row (BKB bytes)
  static constexpr int LDR = BK + 16 / (int)sizeof(T);
  static constexpr int RV = BKB / 16;               // 16-byte vectors per staged row
  static constexpr int NT = 64 * WM * WN;  // threads per workgroup
  static constexpr int TM = BM / WM / 16, TN = BN / WN / 16;
  static_assert(TM >= 1 && TN >= 1, "wave tile must hold a 16x16 block");

  // ALL: all fragments of the staged k tile are read before its MFMAs (one
  // LDS wait per tile); otherwise one k group at a time (fewer registers).
  template <bool ALL = true>
  __device__ static __forceinline__ void compute(f32x4_t (&acc)[TM][TN], const T *As, const T *Bs,
                                                 int wm0, int wn0, int lane) {
    const int li = lane & 15, lg = lane >> 4;
    constexpr int KG = BK / 32;
    if constexpr (!ALL) {
#pragma unroll
      for (int kg = 0; kg < KG; ++kg) {
        Frag<T> a[TM], b[TN];
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) load_frag(a[tm], As + (wm0 + tm * 16 + li) * LDR + kg * 32 + lg * 8);
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) load_frag(b[tn], Bs + (wn0 + tn * 16 + li) * LDR + kg * 32 + lg * 8);
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
          for (int tn = 0; tn < TN; ++tn) mma(acc[tm][tn], a[tm], b[tn]);
      }
      return;
    }
    Frag<T> a[KG][TM], b[KG][TN];
#pragma unroll
    for (int kg = 0; kg < KG; ++kg) {
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) load_frag(a[kg][tm], As + (wm0 + tm * 16 + li) * LDR + kg * 32 + lg * 8);
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) load_frag(b[kg][tn], Bs + (wn0 + tn * 16 + li) * LDR + kg * 32 + lg * 8);
    }
#pragma unroll
    for (int kg = 0; kg < KG; ++kg)
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) mma(acc[tm][tn], a[kg][tm], b[kg][tn]);
  }
};

// ------------------------------------------------------ forward / dgrad
template <typename T, int BM, int BN, int WM, int WN, bool VA, int EPI, int DEPTH, int BKB, int OCC>
__global__ void __launch_bounds__(64 * WM * WN) __attribute__((amdgpu_waves_per_eu(OCC)))
conv_kernel(ConvArgs a, FastDiv fd_w, FastDiv fd_h, FastDiv fd_c, int MT, int NT) {
  using E = ElemT<T>;
  using TL = Tile<T, BM, BN, WM, WN, BKB>;
  constexpr int VEC = TL::VEC, BK = TL::BK, LDR = TL::LDR;
  constexpr int RV = TL::RV;
  constexpr int RP = TL::NT / RV;  // tile rows loaded per pass
  constexpr int AV = (BM + RP - 1) / RP, BV = (BN + RP - 1) / RP;  // last pass may be partial
  __shared__ __attribute__((aligned(16))) T As[2][BM * LDR];
  __shared__ __attribute__((aligned(16))) T Bs[2][BN * LDR];

  const int tid = threadIdx.x;
  // tile coordinates are workgroup-uniform: keep them in scalar registers
  const uint32_t t = xcd_swizzle(blockIdx.x, (uint32_t)(MT * NT * a.C));
  const int nt = __builtin_amdgcn_readfirstlane((int)(t % (uint32_t)NT));
  const uint32_t rest = t / (uint32_t)NT;
  const int mt = __builtin_amdgcn_readfirstlane((int)(rest % (uint32_t)MT));
  const int rep = replica_of(a.rmap, __builtin_amdgcn_readfirstlane((int)(rest / (uint32_t)MT)));
  const int M = a.Bt * a.H * a.W;
  const int m0 = mt * BM, n0 = nt * BN;
  const T *src = reinterpret_cast<const T *>(a.src) + rep * a.src_rs;
  const T *wt = reinterpret_cast<const T *>(a.wt) + rep * a.wt_rs;

  const int kv = tid % RV, rrow = tid / RV;
  int ab[AV], ah[AV], aw[AV];
  bool aok[AV];
  // Vector path: byte offset of each A row's centre pixel and the 9-bit mask
  // of kernel taps that stay inside the image; B rows' byte offsets.
  uint32_t rowoff[AV], tapmask[AV], offb[BV];
  constexpr uint32_t ESZ = sizeof(T);
#pragma unroll
  for (int j = 0; j < AV; ++j) {
    const int m = m0 + rrow + RP * j;
    aok[j] = m < M && (BM % RP == 0 || rrow + RP * j < BM);
    const uint32_t mm = aok[j] ? (uint32_t)m : 0u;
    const uint32_t q = fdiv(mm, fd_w);
    aw[j] = (int)(mm - q * (uint32_t)a.W);
    ab[j] = (int)fdiv(q, fd_h);
    ah[j] = (int)(q - (uint32_t)ab[j] * (uint32_t)a.H);
    if constexpr (VA) {
      rowoff[j] = (uint32_t)mm * (uint32_t)a.Csrc * ESZ;
      uint32_t mk = 0;
#pragma unroll
      for (int rs = 0; rs < 9; ++rs) {
        const int hh = ah[j] + rs / 3 - 1, ww = aw[j] + rs % 3 - 1;
        if ((unsigned)hh < (unsigned)a.H && (unsigned)ww < (unsigned)a.W) mk |= 1u << rs;
      }
      tapmask[j] = aok[j] ? mk : 0u;
    }
  }
#pragma unroll
  for (int j = 0; j < BV; ++j) {
    const int n = n0 + rrow + RP * j;
    offb[j] = (n < a.N && (BN % RP == 0 || rrow + RP * j < BN))
                  ? ((uint32_t)n * (uint32_t)a.Kp + (uint32_t)(kv * VEC)) * ESZ
                  : kOob;
  }
  const __amdgpu_buffer_rsrc_t rsa = make_rsrc(src, (uint32_t)(a.src_rs * ESZ));
  const __amdgpu_buffer_rsrc_t rsb = make_rsrc(wt, (uint32_t)((int64_t)a.N * a.Kp * ESZ));

  // DEPTH register sets: with two, tile kt+2 is fetched while tile kt is
  // multiplied, so each global load has two k tiles of work to arrive in.
  uint4 ra0[AV], rb0[BV], ra1[DEPTH == 2 ? AV : 1], rb1[DEPTH == 2 ? BV : 1];
  auto load_tiles = [&](int kt, uint4 (&ra)[AV], uint4 (&rb)[BV]) {
    const int k0 = kt * BK + kv * VEC;
    if constexpr (VA) {
      // tap (r, s) and channel of this thread's 16-byte vector (im2col rows:
      // the centre tap, channel k0)
      const int rs = a.taps == 1 ? 4 : (int)fdiv((uint32_t)k0, fd_c);
      const int c = k0 - (a.taps == 1 ? 0 : rs * a.Csrc);
      const int r = (rs * 11) >> 5;  // rs / 3 for rs < 9
      const int tap = ((r - 1) * a.W + (rs - 3 * r - 1)) * a.Csrc + c;
      const uint32_t live = k0 < a.K ? 1u : 0u;
#pragma unroll
      for (int j = 0; j < AV; ++j) {
        const bool ok = ((tapmask[j] >> rs) & live) != 0u;
        ra[j] = buffer_load16(rsa, ok ? rowoff[j] + (uint32_t)(tap * (int)ESZ) : kOob, 0);
      }
    } else {
#pragma unroll
      for (int j = 0; j < AV; ++j) {
        Pack<T> pk;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const int k = k0 + e;
          T v = T(0);
          if (k < a.K && aok[j]) {
            const int rs = (int)fdiv((uint32_t)k, fd_c);
            const int c = k - rs * a.Csrc;
            const int r = (rs * 11) >> 5, s = rs - 3 * r;
            const int hh = ah[j] + r - 1, ww = aw[j] + s - 1;
            if ((unsigned)hh < (unsigned)a.H && (unsigned)ww < (unsigned)a.W)
              v = src[((int64_t)(ab[j] * a.H + hh) * a.W + ww) * a.Csrc + c];
          }
          pk.v[e] = v;
        }
        ra[j] = __builtin_bit_cast(uint4, pk);
      }
    }
#pragma unroll
    for (int j = 0; j < BV; ++j) rb[j] = buffer_load16(rsb, offb[j], (uint32_t)(kt * BK) * ESZ);
  };
  auto store_tiles = [&](int buf, const uint4 (&ra)[AV], const uint4 (&rb)[BV]) {
#pragma unroll
    for (int j = 0; j < AV; ++j)
      if (BM % RP == 0 || rrow + RP * j < BM)
        *reinterpret_cast<uint4 *>(&As[buf][(rrow + RP * j) * LDR + kv * VEC]) = ra[j];
#pragma unroll
    for (int j = 0; j < BV; ++j)
      if (BN % RP == 0 || rrow + RP * j < BN)
        *reinterpret_cast<uint4 *>(&Bs[buf][(rrow + RP * j) * LDR + kv * VEC]) = rb[j];
  };

  const int lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave / WN) * (BM / WM), wn0 = (wave % WN) * (BN / WN);
  f32x4_t acc[TL::TM][TL::TN];
#pragma unroll
  for (int i = 0; i < TL::TM; ++i)
#pragma unroll
    for (int j = 0; j < TL::TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int nk = a.Kp / BK;
  if constexpr (DEPTH == 2) {
    load_tiles(0, ra0, rb0);
    if (nk > 1) load_tiles(1, ra1, rb1);
    store_tiles(0, ra0, rb0);
    __syncthreads();
    for (int kt = 0; kt < nk; kt += 2) {
      if (kt + 2 < nk) load_tiles(kt + 2, ra0, rb0);
      TL::compute(acc, As[0], Bs[0], wm0, wn0, lane);
      if (kt + 1 < nk) store_tiles(1, ra1, rb1);
      __syncthreads();
      if (kt + 1 < nk) {
        if (kt + 3 < nk) load_tiles(kt + 3, ra1, rb1);
        TL::compute(acc, As[1], Bs[1], wm0, wn0, lane);
        if (kt + 2 < nk) store_tiles(0, ra0, rb0);
        __syncthreads();
      }
    }
  } else {
    load_tiles(0, ra0, rb0);
    store_tiles(0, ra0, rb0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      const int buf = kt & 1;
      if (kt + 1 < nk) load_tiles(kt + 1, ra0, rb0);
      TL::compute(acc, As[buf], Bs[buf], wm0, wn0, lane);
      if (kt + 1 < nk) store_tiles(buf ^ 1, ra0, rb0);
      __syncthreads();
    }
  }

  // epilogue
  const int li = lane & 15, lg = lane >> 4;
  T *out = reinterpret_cast<T *>(a.out) + rep * a.out_rs;
  const T *res = a.res ? reinterpret_cast<const T *>(a.res) + rep * a.out_rs : nullptr;
  const T *msk = a.mask ? reinterpret_cast<const T *>(a.mask) + rep * a.out_rs : nullptr;
#pragma unroll
  for (int tn = 0; tn < TL::TN; ++tn) {
    const int n = n0 + wn0 + tn * 16 + li;
    const bool nok = n < a.N;
    const float bias = (EPI == EPI_FWD && nok) ? a.bias[rep * a.bias_rs + n] : 0.f;
#pragma unroll
    for (int tm = 0; tm < TL::TM; ++tm) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm0 + tm * 16 + lg * 4 + r;
        if (m < M && nok) {
          const int64_t o = (int64_t)m * a.N + n;
          float v = acc[tm][tn][r];
          if constexpr (EPI == EPI_FWD) {
            v += bias;
            if (res) v += E::to_f(res[o]);
            if (!a.no_relu) v = fmaxf(v, 0.f);
          } else {
            if (res) v += E::to_f(res[o]);
            if (msk && !(E::to_f(msk[o]) > 0.f)) v = 0.f;
          }
          out[o] = E::from_f(v);
        }
      }
    }
  }
}

// --------------------------------------------------------------- wgrad
template <typename T>
__device__ __forceinline__ void transpose_block(const uint4 (&in)[ElemT<T>::VEC],
                                                uint4 (&out)[ElemT<T>::VEC]);

// 8 pixels x 8 bf16 channels -> 8 channels x 8 pixels.
template <>
__device__ __forceinline__ void transpose_block<bf16_t>(const uint4 (&in)[8], uint4 (&out)[8]) {
  uint32_t w[8][4];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    w[e][0] = in[e].x; w[e][1] = in[e].y; w[e][2] = in[e].z; w[e][3] = in[e].w;
  }
  // word j of output row q packs channel q of pixels 2j (low half) and 2j+1
  // (high half): one byte permute per word
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    uint32_t o[4];
    const int wi = q >> 1;
    const uint32_t sel = (q & 1) ? 0x07060302u : 0x05040100u;
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] = __builtin_amdgcn_perm(w[2 * j + 1][wi], w[2 * j][wi], sel);
    out[q] = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

// 4 pixels x 4 fp32 channels -> 4 channels x 4 pixels.
template <>
__device__ __forceinline__ void transpose_block<float>(const uint4 (&in)[4], uint4 (&out)[4]) {
  out[0] = make_uint4(in[0].x, in[1].x, in[2].x, in[3].x);
  out[1] = make_uint4(in[0].y, in[1].y, in[2].y, in[3].y);
  out[2] = make_uint4(in[0].z, in[1].z, in[2].z, in[3].z);
  out[3] = make_uint4(in[0].w, in[1].w, in[2].w, in[3].w);
}

// Transpose a VEC x VEC (pixel x channel) block and store channel row q at
// dst + q * ldr, one row at a time (keeps few registers live).
template <typename T>
__device__ __forceinline__ void store_transposed(const uint4 (&in)[ElemT<T>::VEC], T *dst, int ldr);

template <>
__device__ __forceinline__ void store_transposed<bf16_t>(const uint4 (&in)[8], bf16_t *dst, int ldr) {
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const uint32_t sel = (q & 1) ? 0x07060302u : 0x05040100u;
    uint32_t o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint4 &lo4 = in[2 * j], &hi4 = in[2 * j + 1];
      const uint32_t lo = (q >> 1) == 0 ? lo4.x : (q >> 1) == 1 ? lo4.y : (q >> 1) == 2 ? lo4.z : lo4.w;
      const uint32_t hi = (q >> 1) == 0 ? hi4.x : (q >> 1) == 1 ? hi4.y : (q >> 1) == 2 ? hi4.z : hi4.w;
      o[j] = __builtin_amdgcn_perm(hi, lo, sel);
    }
    *reinterpret_cast<uint4 *>(dst + q * ldr) = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

template <>
__device__ __forceinline__ void store_transposed<float>(const uint4 (&in)[4], float *dst, int ldr) {
  uint4 o[4];
  transpose_block<float>(in, o);
#pragma unroll
  for (int q = 0; q < 4; ++q) *reinterpret_cast<uint4 *>(dst + q * ldr) = o[q];
}

template <typename T, int BM, int BN, int WM, int WN, bool VB>
__global__ void __launch_bounds__(64 * WM * WN) __attribute__((amdgpu_waves_per_eu(WM * WN >= 8 ? 4 : 2)))
wgrad_kernel(WgradArgs a, FastDiv fd_w, FastDiv fd_h, FastDiv fd_c, int MT, int NT) {
  using TL = Tile<T, BM, BN, WM, WN>;
  constexpr int VEC = TL::VEC, BK = TL::BK, LDR = TL::LDR;
  constexpr int NTH = TL::NT;
  constexpr int PB = BK / VEC;  // pixel blocks per k tile
  constexpr int NA = (BM / VEC) * PB, NB = (BN / VEC) * PB;
  constexpr int ITER = (NA + NB + NTH - 1) / NTH;
  static_assert(NA <= NTH, "A blocks must fit one pass");
  __shared__ __attribute__((aligned(16))) T As[2][BM * LDR];
  __shared__ __attribute__((aligned(16))) T Bs[2][BN * LDR];
  __shared__ float red[PB][BM];

  const int tid = threadIdx.x;
  const uint32_t total = (uint32_t)(MT * NT * a.splits * a.C);
  const uint32_t t = xcd_swizzle(blockIdx.x, total);
  const int nt = __builtin_amdgcn_readfirstlane((int)(t % (uint32_t)NT));
  uint32_t rest = t / (uint32_t)NT;
  const int mt = __builtin_amdgcn_readfirstlane((int)(rest % (uint32_t)MT));
  rest /= (uint32_t)MT;
  const int split = __builtin_amdgcn_readfirstlane((int)(rest % (uint32_t)a.splits));
  const int rep = replica_of(a.rmap, __builtin_amdgcn_readfirstlane((int)(rest / (uint32_t)a.splits)));
  const int M = a.Bt * a.H * a.W;
  const int NW = a.taps == 1 ? a.Ci : 9 * a.Ci;  // columns of the (padded) im2col operand
  const int p_begin = split * a.chunk;
  const int p_end = min(M, p_begin + a.chunk);
  const int nk = (p_end - p_begin + BK - 1) / BK;
  const int m0 = mt * BM, n0 = nt * BN;
  const T *G = reinterpret_cast<const T *>(a.g) + rep * a.g_rs;
  const T *X = reinterpret_cast<const T *>(a.x) + rep * a.x_rs;
  const bool do_bias = (nt == 0) && a.db != nullptr;

  // blocks owned by this thread
  int kind[ITER], rowb[ITER], pb[ITER], br[ITER], bs[ITER], bc[ITER];
  bool bvalid[ITER];
#pragma unroll
  for (int it = 0; it < ITER; ++it) {
    const int i = tid + NTH * it;
    if (i < NA) {
      kind[it] = 0;
      rowb[it] = i / PB;
      pb[it] = i % PB;
    } else if (i < NA + NB) {
      kind[it] = 1;
      rowb[it] = (i - NA) / PB;
      pb[it] = (i - NA) % PB;
    } else {
      kind[it] = 2;
      rowb[it] = 0;
      pb[it] = 0;
    }
    br[it] = bs[it] = bc[it] = 0;
    bvalid[it] = false;
    if (kind[it] == 1) {
      const int kk0 = n0 + rowb[it] * VEC;
      bvalid[it] = kk0 < NW;
      if (VB && bvalid[it]) {
        const int rs = a.taps == 1 ? 4 : (int)fdiv((uint32_t)kk0, fd_c);
        bc[it] = kk0 - (a.taps == 1 ? 0 : rs * a.Ci);
        br[it] = (rs * 11) >> 5;
        bs[it] = rs - 3 * br[it];
      }
    }
  }

  // DEPTH register sets of prefetched blocks (tile kt + DEPTH is in flight
  // while tile kt is multiplied).
  constexpr int DEPTH = WM * WN >= 8 ? 1 : 2;
  uint4 reg0[ITER][VEC], reg1[DEPTH == 2 ? ITER : 1][VEC];
  float bsum[VEC];
#pragma unroll
  for (int q = 0; q < VEC; ++q) bsum[q] = 0.f;

  // Gradient rows: contiguous pixels, so one buffer offset per pixel; pixels
  // past the tensor read zero.  Input rows (vector path, W % VEC == 0): a
  // block's VEC pixels share (b, h), only its first or last pixel can leave
  // the image row for kernel column s = 0 or 2.
  constexpr uint32_t ESZ = sizeof(T);
  const __amdgpu_buffer_rsrc_t rsg = make_rsrc(G, (uint32_t)((int64_t)M * a.Co * ESZ));
  const __amdgpu_buffer_rsrc_t rsx = make_rsrc(X, (uint32_t)((int64_t)M * a.Ci * ESZ));
  auto load_tiles = [&](int kt, auto &reg) {
#pragma unroll
    for (int it = 0; it < ITER; ++it) {
      const int pbase = p_begin + kt * BK + pb[it] * VEC;
      if (kind[it] == 0) {
        const int c0 = m0 + rowb[it] * VEC;
        const uint32_t o0 = c0 < a.Co ? ((uint32_t)pbase * (uint32_t)a.Co + (uint32_t)c0) * ESZ : kOob;
#pragma unroll
        for (int e = 0; e < VEC; ++e) reg[it][e] = buffer_load16(rsg, o0 + (uint32_t)(e * a.Co) * ESZ, 0);
        continue;
      }
      if constexpr (VB) {
        if (kind[it] == 1 && a.taps == 1) {
          // im2col rows: contiguous pixels, like the gradient operand
          const uint32_t o0 = bvalid[it] ? ((uint32_t)pbase * (uint32_t)a.Ci + (uint32_t)bc[it]) * ESZ : kOob;
#pragma unroll
          for (int e = 0; e < VEC; ++e) reg[it][e] = buffer_load16(rsx, o0 + (uint32_t)(e * a.Ci) * ESZ, 0);
        } else if (kind[it] == 1) {
          const uint32_t q1 = fdiv((uint32_t)pbase, fd_w);
          const int w0 = (int)((uint32_t)pbase - q1 * (uint32_t)a.W);
          const int b = (int)fdiv(q1, fd_h);
          const int h = (int)(q1 - (uint32_t)b * (uint32_t)a.H);
          const int hh = h + br[it] - 1;
          const bool rowok = bvalid[it] && pbase < M && (unsigned)hh < (unsigned)a.H;
          const int base = ((b * a.H + hh) * a.W + w0 + bs[it] - 1) * a.Ci + bc[it];
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            bool ok = rowok;
            if (e == 0) ok = ok && (w0 + bs[it] - 1 >= 0);
            if (e == VEC - 1) ok = ok && (w0 + VEC - 1 + bs[it] - 1 < a.W);
            reg[it][e] = buffer_load16(rsx, ok ? (uint32_t)(base + e * a.Ci) * ESZ : kOob, 0);
          }
        } else {
#pragma unroll
          for (int e = 0; e < VEC; ++e) reg[it][e] = make_uint4(0, 0, 0, 0);
        }
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const int p = pbase + e;
          uint4 v = make_uint4(0, 0, 0, 0);
          if (kind[it] == 1 && p < p_end && bvalid[it]) {
            const uint32_t q1 = fdiv((uint32_t)p, fd_w);
            const int w = (int)((uint32_t)p - q1 * (uint32_t)a.W);
            const int b = (int)fdiv(q1, fd_h);
            const int h = (int)(q1 - (uint32_t)b * (uint32_t)a.H);
            Pack<T> pk;
            const int kk0 = n0 + rowb[it] * VEC;
#pragma unroll
            for (int q = 0; q < VEC; ++q) {
              const int kk = kk0 + q;
              T val = T(0);
              if (kk < NW) {
                const int rs = (int)fdiv((uint32_t)kk, fd_c);
                const int c = kk - rs * a.Ci;
                const int r = (rs * 11) >> 5, s = rs - 3 * r;
                const int hh = h + r - 1, ww = w + s - 1;
                if ((unsigned)hh < (unsigned)a.H && (unsigned)ww < (unsigned)a.W)
                  val = X[((int64_t)(b * a.H + hh) * a.W + ww) * a.Ci + c];
              }
              pk.v[q] = val;
            }
            v = __builtin_bit_cast(uint4, pk);
          }
          reg[it][e] = v;
        }
      }
    }
  };
  auto store_tiles = [&](int buf, auto &reg) {
#pragma unroll
    for (int it = 0; it < ITER; ++it) {
      if (kind[it] == 2) continue;
      if (kind[it] == 0 && do_bias) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          Pack<T> p = __builtin_bit_cast(Pack<T>, reg[it][e]);
#pragma unroll
          for (int q = 0; q < VEC; ++q) bsum[q] += ElemT<T>::to_f(p.v[q]);
        }
      }
      T *dst = kind[it] == 0 ? As[buf] : Bs[buf];
      store_transposed<T>(reg[it], dst + rowb[it] * VEC * LDR + pb[it] * VEC, LDR);
    }
  };

  const int lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave / WN) * (BM / WM), wn0 = (wave % WN) * (BN / WN);
  f32x4_t acc[TL::TM][TL::TN];
#pragma unroll
  for (int i = 0; i < TL::TM; ++i)
#pragma unroll
    for (int j = 0; j < TL::TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  if constexpr (DEPTH == 2) {
    if (nk > 0) {
      load_tiles(0, reg0);
      if (nk > 1) load_tiles(1, reg1);
      store_tiles(0, reg0);
    }
    __syncthreads();
    for (int kt = 0; kt < nk; kt += 2) {
      if (kt + 2 < nk) load_tiles(kt + 2, reg0);
      TL::template compute<false>(acc, As[0], Bs[0], wm0, wn0, lane);
      if (kt + 1 < nk) store_tiles(1, reg1);
      __syncthreads();
      if (kt + 1 < nk) {
        if (kt + 3 < nk) load_tiles(kt + 3, reg1);
        TL::template compute<false>(acc, As[1], Bs[1], wm0, wn0, lane);
        if (kt + 2 < nk) store_tiles(0, reg0);
        __syncthreads();
      }
    }
  } else {
    if (nk > 0) {
      load_tiles(0, reg0);
      store_tiles(0, reg0);
    }
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      const int buf = kt & 1;
      if (kt + 1 < nk) load_tiles(kt + 1, reg0);
      TL::template compute<false>(acc, As[buf], Bs[buf], wm0, wn0, lane);
      if (kt + 1 < nk) store_tiles(buf ^ 1, reg0);
      __syncthreads();
    }
  }

  const int li = lane & 15, lg = lane >> 4;
  float *dw = a.dw + split * a.dw_ss + rep * a.dw_rs;
#pragma unroll
  for (int tn = 0; tn < TL::TN; ++tn) {
    const int n = n0 + wn0 + tn * 16 + li;
#pragma unroll
    for (int tm = 0; tm < TL::TM; ++tm)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm0 + tm * 16 + lg * 4 + r;
        if (m < a.Co && n < a.nw) dw[(int64_t)m * a.nw + n] = acc[tm][tn][r];
      }
  }

  if (do_bias) {
    if (kind[0] == 0) {
#pragma unroll
      for (int q = 0; q < VEC; ++q) red[pb[0]][rowb[0] * VEC + q] = bsum[q];
    }
    __syncthreads();
    if (tid < BM) {
      const int co = m0 + tid;
      if (co < a.Co) {
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < PB; ++i) s += red[i][tid];
        a.db[split * a.db_ss + rep * a.db_rs + co] = s;
      }
    }
  }
}

template <typename T> const char *tname() { return sizeof(T) == 2 ? "bf16" : "f32"; }

template <typename T, int BM, int BN, bool VA, int WM = 2, int WN = 2, int DEPTH = 2, int BKB = 128, int OCC = 2>
hipError_t run_conv(const ConvArgs &a, hipStream_t s, std::string *label) {
  const int M = a.Bt * a.H * a.W;
  const int MT = (M + BM - 1) / BM, NT = (a.N + BN - 1) / BN;
  const FastDiv fw = make_fastdiv(a.W), fh = make_fastdiv(a.H), fc = make_fastdiv(a.Csrc);
  const uint32_t blocks = (uint32_t)MT * NT * a.C;
  if (label)
    *label = std::string(a.epi == EPI_FWD ? "conv_fwd<" : "conv_dgrad<") + tname<T>() + "," +
             std::to_string(BM) + "x" + std::to_string(BN) + "x" + std::to_string(BKB / (int)sizeof(T)) + ",w" +
             std::to_string(WM * WN) + (VA ? ",vec>" : ",gather>");
  const dim3 threads(64 * WM * WN);
  if (a.epi == EPI_FWD)
    hipLaunchKernelGGL((conv_kernel<T, BM, BN, WM, WN, VA, EPI_FWD, DEPTH, BKB, OCC>), dim3(blocks), threads, 0, s, a,
                       fw, fh, fc, MT, NT);
  else
    hipLaunchKernelGGL((conv_kernel<T, BM, BN, WM, WN, VA, EPI_DGRAD, DEPTH, BKB, OCC>), dim3(blocks), threads, 0, s,
                       a, fw, fh, fc, MT, NT);
  return hipGetLastError();
}

template <typename T, bool VA>
hipError_t pick_conv(const ConvArgs &a, hipStream_t s, std::string *label) {
  // 16-bit tiles run 8 waves (4 per SIMD at two workgroups per CU): the extra
  // resident waves hide LDS and global latency better than larger wave tiles.
  if constexpr (sizeof(T) == 2) {
    if (a.N > 64) return run_conv<T, 128, 128, VA, 4, 2, 1, 128, 4>(a, s, label);
    if (a.N > 32) return run_conv<T, 128, 64, VA, 4, 2, 1, 128, 4>(a, s, label);
    return run_conv<T, 128, 32, VA, 4, 2, 1, 128, 4>(a, s, label);
  } else {
    if (a.N > 64) return run_conv<T, 128, 128, VA>(a, s, label);
    if (a.N > 32) return run_conv<T, 128, 64, VA>(a, s, label);
    return run_conv<T, 128, 32, VA>(a, s, label);
  }
}

template <typename T, int BM, int BN, bool VB, int WM = 2, int WN = 2>
hipError_t run_wgrad(const WgradArgs &a, hipStream_t s, std::string *label) {
  const int MT = (a.Co + BM - 1) / BM, NT = ((a.taps == 1 ? a.Ci : 9 * a.Ci) + BN - 1) / BN;
  const FastDiv fw = make_fastdiv(a.W), fh = make_fastdiv(a.H), fc = make_fastdiv(a.Ci);
  const uint32_t blocks = (uint32_t)MT * NT * a.splits * a.C;
  if (label)
    *label = std::string("conv_wgrad<") + tname<T>() + "," + std::to_string(BM) + "x" + std::to_string(BN) +
             ",w" + std::to_string(WM * WN) + (VB ? ",vec>" : ",gather>");
  hipLaunchKernelGGL((wgrad_kernel<T, BM, BN, WM, WN, VB>), dim3(blocks), dim3(64 * WM * WN), 0, s, a, fw, fh, fc,
                     MT, NT);
  return hipGetLastError();
}

template <typename T, int BM, bool VB>
hipError_t pick_wgrad_n(const WgradArgs &a, hipStream_t s, std::string *label) {
  const int NW = a.taps == 1 ? a.Ci : 9 * a.Ci;
  if constexpr (sizeof(T) == 2 && BM == 128) {
    if (NW > 64) return run_wgrad<T, BM, 128, VB, 2, 4>(a, s, label);
  }
  if (NW > 64) return run_wgrad<T, BM, 128, VB>(a, s, label);
  if (NW > 32) return run_wgrad<T, BM, 64, VB>(a, s, label);
  return run_wgrad<T, BM, 32, VB>(a, s, label);
}

template <typename T, bool VB>
hipError_t pick_wgrad(const WgradArgs &a, hipStream_t s, std::string *label) {
  int bm, bn;
  wgrad_tile(sizeof(T) == 2 ? GCPSL_BF16 : GCPSL_F32, a.Co, a.taps == 1 ? a.Ci : 9 * a.Ci, &bm, &bn);
  if (bm == 128) return pick_wgrad_n<T, 128, VB>(a, s, label);
  if (bm == 64) return pick_wgrad_n<T, 64, VB>(a, s, label);
  return pick_wgrad_n<T, 32, VB>(a, s, label);
}

}  // namespace

int wgrad_k_tile(int dtype) { return dtype == GCPSL_BF16 ? 64 : 32; }

void wgrad_tile(int dtype, int Co, int ncols, int *bm, int *bn) {
  const int nw = ncols;
  *bm = Co > 64 ? 128 : (Co > 32 ? 64 : 32);
  *bn = nw > 64 ? 128 : (nw > 32 ? 64 : 32);
}

hipError_t launch_conv(int dtype, const ConvArgs &a, hipStream_t s, std::string *label) {
  // routing codes: the head's pooling epilogue (halo tile) and the
  // image-side kernels take them
  if (a.pool_code) {
    if (a.epi == EPI_FWD && a.pool_max && a.pool_out && conv_fuses_avg(dtype, a)) return launch_conv_lds(a, s, label);
    return (conv_pool_codes(dtype, a) && (a.epi == EPI_DGRAD || a.pool_out)) ? launch_conv_img(a, s, label)
                                                                              : hipErrorInvalidValue;
  }
  if (a.taps == 9 && a.epi == EPI_FWD && a.res == nullptr && conv_im3_ok(dtype, a.Csrc, a.N, a.H, a.W))
    return launch_conv_col(a, s, label);
  if (conv_img_ok(dtype, a)) return launch_conv_img(a, s, label);
  if (a.epi == EPI_FWD && conv_col_ok(dtype, a)) return launch_conv_col(a, s, label);
  if (conv_lds_ok(dtype, a)) return launch_conv_lds(a, s, label);
  if (dtype == GCPSL_BF16)
    return (a.Csrc % 8 == 0) ? pick_conv<bf16_t, true>(a, s, label) : pick_conv<bf16_t, false>(a, s, label);
  return (a.Csrc % 4 == 0) ? pick_conv<float, true>(a, s, label) : pick_conv<float, false>(a, s, label);
}

hipError_t launch_wgrad(int dtype, const WgradArgs &a, hipStream_t s, std::string *label) {
  if (a.gcode)
    return (wgrad_pool_codes(dtype, a.Co, a.Ci, a.H, a.W, a.taps) && wgrad_lds_ok(dtype, a.Co, a.Ci) &&
            a.chunk % 64 == 0)
               ? launch_wgrad_lds(a, s, label)
               : hipErrorInvalidValue;
  if ((wgrad_col_ok(dtype, a.Co, a.Ci, a.taps) ||
       (a.taps == 9 && conv_im3_ok(dtype, a.Ci, a.Co, a.H, a.W))) && a.chunk % 128 == 0)
    return launch_wgrad_col(a, s, label);
  if (wgrad_lds_ok(dtype, a.Co, a.Ci) && a.chunk % 64 == 0) return launch_wgrad_lds(a, s, label);
  // vector path: whole 16-byte channel vectors and pixel blocks within one
  // image row (im2col rows need no image-row structure)
  if (dtype == GCPSL_BF16)
    return (a.Ci % 8 == 0 && (a.taps == 1 || a.W % 8 == 0)) ? pick_wgrad<bf16_t, true>(a, s, label)
                                                            : pick_wgrad<bf16_t, false>(a, s, label);
  return (a.Ci % 4 == 0 && (a.taps == 1 || a.W % 4 == 0)) ? pick_wgrad<float, true>(a, s, label)
                                                          : pick_wgrad<float, false>(a, s, label);
}
