// Forward and input-gradient (dgrad) 3x3 convolutions, bf16, on gfx950, as
// implicit GEMMs over k = (r, s, c):
//
//   fwd    out[m][n] = ReLU(sum_k x[m + (r-1, s-1)][c] Wf[n][k] + bias[n] (+ res[m][n]))
//   dgrad  dx[m][n]  = (sum_k g[m + (r-1, s-1)][c] Wd[n][k] (+ res[m][n])) * [mask[m][n] > 0]
//
// (dgrad is a forward conv of g with the flipped, transposed weights Wd).
// Both operands are k-contiguous: a k tile (64 values, 128 bytes per row) of
// 128 pixel rows (gathered per kernel tap from the NHWC activation) and of
// 256 weight rows is copied into LDS by buffer loads that write LDS directly;
// taps outside the image, pixels past the batch and weight rows past N read
// zero through the buffer range check.  Rows are XOR-swizzled in 16-byte
// chunks (chunk ^ ((row >> 1) & 7)) so that the 16 rows of one fragment read
// hit all banks.  Three LDS stages rotate; the fragment reads are inline asm
// with explicit lgkmcnt waits so the compiler does not wait for every
// outstanding copy, and the k loop is software-pipelined so that MFMAs
// cover the LDS latency across the per-tile barrier.
//
// The MFMA takes weight fragments as its A operand and pixel fragments as B,
// so each lane accumulates 4 consecutive output channels of one pixel.  The
// epilogue stages the fp32 tile through LDS and then works on 8 consecutive
// channels per lane: 16-byte loads of the residual and mask, 16-byte stores.
//
// Workgroup: 8 waves, 128 pixels x 256 output channels, 64 x 64 per wave.
#include "runtime.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#define LDS_PTR(p) ((__attribute__((address_space(3))) void *)(p))

constexpr int BM = 128, BN = 256, BK = 64, NS = 3, NTHR = 512;
constexpr int ROW = BK * 2;  // bytes per LDS row
constexpr int A_BYTES = BM * ROW, B_BYTES = BN * ROW;
constexpr int STAGE = A_BYTES + B_BYTES;
constexpr int SA = A_BYTES / (NTHR * 16), SB = B_BYTES / (NTHR * 16);
constexpr int LDS_BYTES = NS * STAGE;
constexpr int EP_LD = 68;  // floats per staged epilogue row (64 + 4 padding)
constexpr uint32_t kOob = 0x80000000u;
constexpr int kBufferFlags = 0x00020000;
static_assert(SA * NTHR * 16 == A_BYTES && SB * NTHR * 16 == B_BYTES, "copies must tile the stage");
static_assert(8 * 64 * EP_LD * 4 <= LDS_BYTES, "epilogue staging must fit the stages");

__device__ __forceinline__ int swz(int row) { return (row >> 1) & 7; }

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *base, uint32_t bytes) {
  const uint64_t p = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)p);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(p >> 32));
  void *q = reinterpret_cast<void *>(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(q, (short)0, (int)__builtin_amdgcn_readfirstlane(bytes), kBufferFlags);
}

__device__ __forceinline__ void mma(f32x4_t &acc, const u32x4 &a, const u32x4 &b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                acc, 0, 0, 0);
}

// Four fragments 16 rows (2048 bytes) apart.
__device__ __forceinline__ void read4(u32x4 (&f)[4], uint32_t addr) {
  asm volatile(
      "ds_read_b128 %0, %4\n\t"
      "ds_read_b128 %1, %4 offset:2048\n\t"
      "ds_read_b128 %2, %4 offset:4096\n\t"
      "ds_read_b128 %3, %4 offset:6144"
      : "=&v"(f[0]), "=&v"(f[1]), "=&v"(f[2]), "=&v"(f[3])
      : "v"(addr));
}

__device__ __forceinline__ void wait_lds(u32x4 (&x)[4], u32x4 (&w)[4]) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(x[0]), "+v"(x[1]), "+v"(x[2]), "+v"(x[3]), "+v"(w[0]), "+v"(w[1]), "+v"(w[2]), "+v"(w[3]));
}

// The 16 MFMAs of one k group (32 values): weight fragments w, pixel fragments x.
__device__ __forceinline__ void mfma_group(f32x4_t (&acc)[4][4], const u32x4 (&x)[4], const u32x4 (&w)[4]) {
#pragma unroll
  for (int tm = 0; tm < 4; ++tm)
#pragma unroll
    for (int tn = 0; tn < 4; ++tn) mma(acc[tm][tn], w[tn], x[tm]);
}

__device__ __forceinline__ float bf2f(uint32_t bits16) { return bf16_to_f32((bf16_t)bits16); }
__device__ __forceinline__ uint32_t f2bf(float f) { return (uint32_t)f32_to_bf16(f); }

template <int EPI, bool TAPS1>
__global__ void __launch_bounds__(NTHR)
conv_lds_kernel(ConvArgs a, FastDiv fd_w, FastDiv fd_h, FastDiv fd_c, int MT, int NT) {
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t t = xcd_swizzle(blockIdx.x, (uint32_t)(MT * NT * a.C));
  const int nt = __builtin_amdgcn_readfirstlane((int)(t % (uint32_t)NT));
  const uint32_t rest = t / (uint32_t)NT;
  const int mt = __builtin_amdgcn_readfirstlane((int)(rest % (uint32_t)MT));
  const int rep = __builtin_amdgcn_readfirstlane((int)(rest / (uint32_t)MT));
  const int M = a.Bt * a.H * a.W;
  const int m0 = mt * BM, n0 = nt * BN;
  const bf16_t *src = reinterpret_cast<const bf16_t *>(a.src) + rep * a.src_rs;
  const bf16_t *wt = reinterpret_cast<const bf16_t *>(a.wt) + rep * a.wt_rs;
  const __amdgpu_buffer_rsrc_t rsa = rsrc(src, (uint32_t)(a.src_rs * 2));
  const __amdgpu_buffer_rsrc_t rsb = rsrc(wt, (uint32_t)((int64_t)a.N * a.Kp * 2));

  // This thread's copies: byte q*8192 + wave*1024 + lane*16 of the A (pixel)
  // and B (weight) regions of a stage.  Row and swizzled chunk are fixed;
  // the k tile advances.
  int achunk[SA], arowoff[SA];
  uint32_t amask[SA];  // kernel taps (bit r*3+s) whose source pixel is inside the image
#pragma unroll
  for (int q = 0; q < SA; ++q) {
    const int byte = q * NTHR * 16 + wave * 1024 + lane * 16;
    const int row = byte / ROW;
    achunk[q] = ((byte % ROW) / 16) ^ swz(row);
    const int m = m0 + row;
    const uint32_t mm = m < M ? (uint32_t)m : 0u;
    arowoff[q] = (int)mm * a.Csrc;
    if constexpr (TAPS1) {
      amask[q] = m < M ? 1u : 0u;
    } else {
      const uint32_t q1 = fdiv(mm, fd_w);
      const int w = (int)(mm - q1 * (uint32_t)a.W);
      const int h = (int)(q1 - fdiv(q1, fd_h) * (uint32_t)a.H);
      uint32_t mk = 0;
#pragma unroll
      for (int rs = 0; rs < 9; ++rs) {
        const int hh = h + rs / 3 - 1, ww = w + rs % 3 - 1;
        if ((unsigned)hh < (unsigned)a.H && (unsigned)ww < (unsigned)a.W) mk |= 1u << rs;
      }
      amask[q] = m < M ? mk : 0u;
    }
  }
  uint32_t boff[SB];
#pragma unroll
  for (int q = 0; q < SB; ++q) {
    const int byte = q * NTHR * 16 + wave * 1024 + lane * 16;
    const int row = byte / ROW;
    const int n = n0 + row;
    boff[q] = n < a.N ? ((uint32_t)n * (uint32_t)a.Kp + (uint32_t)(8 * (((byte % ROW) / 16) ^ swz(row)))) * 2u
                      : kOob;
  }

  // Tile kt >= nk is never multiplied; its copies only keep the count of
  // copies in flight uniform (their stage is free by then: no reads follow).
  const int nk = a.Kp / BK;
  char *stage0 = smem + wave * 1024;
  auto issue = [&](int kt) {
    char *sa = stage0 + (kt % NS) * STAGE;
#pragma unroll
    for (int q = 0; q < SA; ++q) {
      const int k = kt * BK + 8 * achunk[q];
      uint32_t off;
      if constexpr (TAPS1) {
        off = ((amask[q] != 0u) & (k < a.K)) ? (uint32_t)(arowoff[q] + k) * 2u : kOob;
      } else {
        // k past K has rs >= 9, outside the mask
        const int rs = (int)fdiv((uint32_t)k, fd_c);
        const int c = k - rs * a.Csrc;
        const int r = (rs * 11) >> 5;  // rs / 3 for rs < 9
        const int tap = ((r - 1) * a.W + (rs - 3 * r - 1)) * a.Csrc + c;
        off = ((amask[q] >> min(rs, 31)) & 1u) ? (uint32_t)(arowoff[q] + tap) * 2u : kOob;
      }
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsa, LDS_PTR(sa + q * NTHR * 16), 16, off, 0, 0, 0);
    }
    const uint32_t kb = kt < nk ? (uint32_t)(kt * BK * 2) : kOob;
#pragma unroll
    for (int q = 0; q < SB; ++q)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsb, LDS_PTR(sa + A_BYTES + q * NTHR * 16), 16,
                                               boff[q] == kOob ? kOob : boff[q] + kb, 0, 0, 0);
  };

  // fragment read addresses: lane (li, lg) reads row li of a 16-row block,
  // chunk 4*kg + lg; rows of one wave's blocks are 16 apart (2048 bytes)
  const int li = lane & 15, lg = lane >> 4;
  const int wm = wave >> 2, wn = wave & 3;
  const uint32_t lds0 = (uint32_t)(size_t)LDS_PTR(smem);
  uint32_t xa[2], wa[2];
#pragma unroll
  for (int kg = 0; kg < 2; ++kg) {
    const int ph = ((4 * kg + lg) ^ swz(li)) * 16;
    xa[kg] = (uint32_t)((wm * 64 + li) * ROW + ph);
    wa[kg] = (uint32_t)(A_BYTES + (wn * 64 + li) * ROW + ph);
  }

  f32x4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[i][k] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Software pipeline over k tiles (R0/R1: fragments of k groups 0/1):
  //   wait R0; read R1; MFMA R0; wait R1       -- this tile's reads are done
  //   wait own copies of tile kt+1; barrier    -- kt+1 visible, stage kt free
  //   copy tile kt+3 into stage kt; read R0 of tile kt+1; MFMA R1
  // so the last 16 MFMAs of a tile cover the next tile's first LDS reads.
  issue(0);
  issue(1);
  issue(2);
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * (SA + SB)) : "memory");
  asm volatile("s_barrier" ::: "memory");
  u32x4 x0[4], w0[4], x1[4], w1[4];
  read4(x0, lds0 + xa[0]);
  read4(w0, lds0 + wa[0]);
  for (int kt = 0; kt < nk; ++kt) {
    const uint32_t st = lds0 + (uint32_t)((kt % NS) * STAGE);
    wait_lds(x0, w0);
    read4(x1, st + xa[1]);
    read4(w1, st + wa[1]);
    mfma_group(acc, x0, w0);
    wait_lds(x1, w1);
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(SA + SB) : "memory");
    asm volatile("s_barrier" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    issue(kt + 3);
    if (kt + 1 < nk) {
      const uint32_t sn = lds0 + (uint32_t)(((kt + 1) % NS) * STAGE);
      read4(x0, sn + xa[0]);
      read4(w0, sn + wa[0]);
    }
    __builtin_amdgcn_sched_barrier(0);
    mfma_group(acc, x1, w1);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  // epilogue: stage the wave's 64 x 64 fp32 tile as [pixel][channel]
  float *ep = reinterpret_cast<float *>(smem) + wave * 64 * EP_LD;
#pragma unroll
  for (int tm = 0; tm < 4; ++tm)
#pragma unroll
    for (int tn = 0; tn < 4; ++tn)
      *reinterpret_cast<f32x4_t *>(ep + (tm * 16 + li) * EP_LD + tn * 16 + lg * 4) = acc[tm][tn];
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

  const int seg = lane & 7;                      // channels 8*seg .. 8*seg+7 of the wave tile
  const int n = n0 + wn * 64 + 8 * seg;
  if (n >= a.N) return;
  float bias[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) bias[e] = EPI == EPI_FWD ? a.bias[rep * a.bias_rs + n + e] : 0.f;
  bf16_t *out = reinterpret_cast<bf16_t *>(a.out) + rep * a.out_rs;
  const bf16_t *res = a.res ? reinterpret_cast<const bf16_t *>(a.res) + rep * a.out_rs : nullptr;
  const bf16_t *msk = a.mask ? reinterpret_cast<const bf16_t *>(a.mask) + rep * a.out_rs : nullptr;
#pragma unroll 2
  for (int i = 0; i < 8; ++i) {
    const int r = (lane >> 3) + 8 * i;  // pixel row of the wave tile
    const int m = m0 + wm * 64 + r;
    if (m >= M) break;
    const f32x4_t lo = *reinterpret_cast<const f32x4_t *>(ep + r * EP_LD + 8 * seg);
    const f32x4_t hi = *reinterpret_cast<const f32x4_t *>(ep + r * EP_LD + 8 * seg + 4);
    float v[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    const int64_t o = (int64_t)m * a.N + n;
    if (res) {
      const uint4 rv = *reinterpret_cast<const uint4 *>(res + o);
      const uint32_t rw[4] = {rv.x, rv.y, rv.z, rv.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[2 * e] += bf2f(rw[e] & 0xffffu);
        v[2 * e + 1] += bf2f(rw[e] >> 16);
      }
    }
    if constexpr (EPI == EPI_FWD) {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = fmaxf(v[e] + bias[e], 0.f);
    } else {
      if (msk) {
        const uint4 mv = *reinterpret_cast<const uint4 *>(msk + o);
        const uint32_t mw[4] = {mv.x, mv.y, mv.z, mv.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (!(bf2f(mw[e] & 0xffffu) > 0.f)) v[2 * e] = 0.f;
          if (!(bf2f(mw[e] >> 16) > 0.f)) v[2 * e + 1] = 0.f;
        }
      }
    }
    uint4 ov;
    ov.x = f2bf(v[0]) | (f2bf(v[1]) << 16);
    ov.y = f2bf(v[2]) | (f2bf(v[3]) << 16);
    ov.z = f2bf(v[4]) | (f2bf(v[5]) << 16);
    ov.w = f2bf(v[6]) | (f2bf(v[7]) << 16);
    *reinterpret_cast<uint4 *>(out + o) = ov;
  }
}

}  // namespace

bool conv_lds_ok(int dtype, const ConvArgs &a) {
  return dtype == GCPSL_BF16 && a.N >= 128 && a.N % 8 == 0 && a.Csrc % 8 == 0 && a.Kp % BK == 0;
}

hipError_t launch_conv_lds(const ConvArgs &a, hipStream_t s, std::string *label) {
  static bool attr = false;
  if (!attr) {
    for (const void *f : {reinterpret_cast<const void *>(&conv_lds_kernel<EPI_FWD, false>),
                          reinterpret_cast<const void *>(&conv_lds_kernel<EPI_FWD, true>),
                          reinterpret_cast<const void *>(&conv_lds_kernel<EPI_DGRAD, false>),
                          reinterpret_cast<const void *>(&conv_lds_kernel<EPI_DGRAD, true>)}) {
      const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, LDS_BYTES);
      if (e != hipSuccess) return e;
    }
    attr = true;
  }
  const int M = a.Bt * a.H * a.W;
  const int MT = (M + BM - 1) / BM, NT = (a.N + BN - 1) / BN;
  const FastDiv fw = make_fastdiv(a.W), fh = make_fastdiv(a.H), fc = make_fastdiv(a.Csrc);
  const uint32_t blocks = (uint32_t)MT * NT * a.C;
  if (label) *label = std::string(a.epi == EPI_FWD ? "conv_fwd" : "conv_dgrad") + "<bf16,128x256x64,w8,lds>";
  const dim3 g(blocks), b(NTHR);
  if (a.epi == EPI_FWD) {
    if (a.taps == 1) hipLaunchKernelGGL((conv_lds_kernel<EPI_FWD, true>), g, b, LDS_BYTES, s, a, fw, fh, fc, MT, NT);
    else hipLaunchKernelGGL((conv_lds_kernel<EPI_FWD, false>), g, b, LDS_BYTES, s, a, fw, fh, fc, MT, NT);
  } else {
    if (a.taps == 1) hipLaunchKernelGGL((conv_lds_kernel<EPI_DGRAD, true>), g, b, LDS_BYTES, s, a, fw, fh, fc, MT, NT);
    else hipLaunchKernelGGL((conv_lds_kernel<EPI_DGRAD, false>), g, b, LDS_BYTES, s, a, fw, fh, fc, MT, NT);
  }
  return hipGetLastError();
}
