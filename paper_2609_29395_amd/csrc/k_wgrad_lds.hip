// Weight and bias gradient of a 3x3 conv layer, bf16, on gfx950:
//
//   dW[co][(r,s,ci)] = sum_p g[p][co] x[p + (r-1, s-1)][ci]      db[co] = sum_p g[p][co]
//
// with p = (b, h, w) running over a chunk of the batch's pixels (split-K).
// Both operands are stored pixel-major (NHWC): the reduction index is the
// outer dimension.  A k tile of 64 pixels is copied into LDS exactly as it
// lies in memory -- 64 rows of 128 output channels (g) and 64 rows of 256
// im2col columns (x, shifted per kernel tap) -- by buffer loads that write LDS
// directly, so no registers stage the tiles and out-of-image taps,
// out-of-chunk pixels and ragged columns are zero-filled by the buffer range
// check.  The MFMA wants each lane to hold 8 consecutive k (pixels) of one
// output row or column; ds_read_b64_tr_b16 produces that from the
// pixel-major tile: within 16 lanes, lane 4r+q reads 4 channels of pixel r
// and lane i receives channel i of the 4 pixels.
//
// LDS rows are XOR-swizzled in 16-byte chunks (chunk ^ swz(row)) so that the
// 16 pixels of one transposing read fall on all banks.  Three LDS stages
// rotate: while tile kt is multiplied the copies of the next two tiles are in
// flight, and tile kt's stage is refilled once every wave has read it.  Each
// wave waits for its own copies (vmcnt), a barrier publishes them.  The LDS
// reads are
// inline asm with explicit lgkmcnt waits so that the compiler does not add a
// wait for every outstanding copy before them, and the k loop is
// software-pipelined so that MFMAs cover the LDS latency across the barrier.
//
// Workgroup: 8 waves, 128 (co) x 256 (columns) outputs, 64 x 64 per wave.
// The bias gradient rides along in the column-tile-0 workgroups: every wave
// multiplies one of its g fragments by a ones fragment (one extra MFMA per
// k group).
#include "runtime.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#define LDS_PTR(p) ((__attribute__((address_space(3))) void *)(p))

constexpr int BM = 128, BN = 256, BK = 64, NS = 3, NTHR = 512;
constexpr int ROWA = BM * 2, ROWB = BN * 2;  // bytes per LDS row
constexpr int A_BYTES = BK * ROWA, B_BYTES = BK * ROWB;
constexpr int STAGE = A_BYTES + B_BYTES;
constexpr int SA = A_BYTES / (NTHR * 16), SB = B_BYTES / (NTHR * 16);  // 16-byte copies per thread
constexpr int LDS_BYTES = NS * STAGE;
constexpr uint32_t kOob = 0x80000000u;
constexpr int kBufferFlags = 0x00020000;
static_assert(SA * NTHR * 16 == A_BYTES && SB * NTHR * 16 == B_BYTES, "copies must tile the stage");
static_assert(SA + SB <= 63, "per-wave copies per tile must fit the vmcnt field");

__device__ __forceinline__ int swz(int row) { return ((row & 3) | ((row >> 1) & 4)) << 1; }

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *base, uint32_t bytes) {
  const uint64_t p = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)p);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(p >> 32));
  void *q = reinterpret_cast<void *>(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(q, (short)0, (int)__builtin_amdgcn_readfirstlane(bytes), kBufferFlags);
}

// One operand fragment: 8 pixels (two transposing reads 4 pixel rows apart).
template <int OFF, int ROW>
__device__ __forceinline__ void read_frag(u32x4 &f, uint32_t addr) {
  u32x2 lo, hi;
  asm volatile("ds_read_b64_tr_b16 %0, %2 offset:%3\n\tds_read_b64_tr_b16 %1, %2 offset:%4"
               : "=&v"(lo), "=&v"(hi)
               : "v"(addr), "n"(OFF), "n"(OFF + 4 * ROW));
  f = __builtin_shufflevector(lo, hi, 0, 1, 2, 3);
}

__device__ __forceinline__ void mma(f32x4_t &acc, const u32x4 &a, const u32x4 &b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                acc, 0, 0, 0);
}

// Fragments of k group G (32 pixels) of the stage at byte address sa: g (A
// operand) and x (B operand); the reads stay in flight until wait_lds.
template <int G>
__device__ __forceinline__ void read_group(u32x4 (&a)[4], u32x4 (&b)[4], const uint32_t (&ra)[4],
                                           const uint32_t (&rb)[4], uint32_t sa) {
#pragma unroll
  for (int i = 0; i < 4; ++i) read_frag<G * 32 * ROWA, ROWA>(a[i], sa + ra[i]);
#pragma unroll
  for (int i = 0; i < 4; ++i) read_frag<G * 32 * ROWB, ROWB>(b[i], sa + rb[i]);
}

__device__ __forceinline__ void wait_lds(u32x4 (&a)[4], u32x4 (&b)[4]) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]), "+v"(b[0]), "+v"(b[1]), "+v"(b[2]), "+v"(b[3]));
}

// The MFMAs of one k group; with bias, the wave's g fragment wn also meets a
// ones fragment (column sums of g).
__device__ __forceinline__ void mfma_group(f32x4_t (&acc)[4][4], f32x4_t &bacc, const u32x4 (&a)[4],
                                           const u32x4 (&b)[4], bool bias, int wn) {
#pragma unroll
  for (int tm = 0; tm < 4; ++tm) {
#pragma unroll
    for (int tn = 0; tn < 4; ++tn) mma(acc[tm][tn], a[tm], b[tn]);
    if (bias && tm == wn) {
      const uint32_t one2 = 0x3F803F80u;  // two bf16 ones
      mma(bacc, a[tm], u32x4{one2, one2, one2, one2});
    }
  }
}

template <bool TAPS1>
__global__ void __launch_bounds__(NTHR)
wgrad_lds_kernel(WgradArgs a, FastDiv fd_w, FastDiv fd_h, FastDiv fd_c, int MT, int NT) {
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t total = (uint32_t)(MT * NT * a.splits * a.C);
  const uint32_t t = xcd_swizzle(blockIdx.x, total);
  const int nt = __builtin_amdgcn_readfirstlane((int)(t % (uint32_t)NT));
  uint32_t rest = t / (uint32_t)NT;
  const int mt = __builtin_amdgcn_readfirstlane((int)(rest % (uint32_t)MT));
  rest /= (uint32_t)MT;
  const int split = __builtin_amdgcn_readfirstlane((int)(rest % (uint32_t)a.splits));
  const int rep = __builtin_amdgcn_readfirstlane((int)(rest / (uint32_t)a.splits));
  const int M = a.Bt * a.H * a.W;
  const int NW = a.taps == 1 ? a.Ci : 9 * a.Ci;
  const int p_begin = split * a.chunk;
  const int p_end = min(M, p_begin + a.chunk);
  const int nk = (p_end - p_begin + BK - 1) / BK;
  const int m0 = mt * BM, n0 = nt * BN;
  const bf16_t *G = reinterpret_cast<const bf16_t *>(a.g) + rep * a.g_rs;
  const bf16_t *X = reinterpret_cast<const bf16_t *>(a.x) + rep * a.x_rs;
  const bool do_bias = (nt == 0) && a.db != nullptr;
  const __amdgpu_buffer_rsrc_t rsg = rsrc(G, (uint32_t)((int64_t)M * a.Co * 2));
  const __amdgpu_buffer_rsrc_t rsx = rsrc(X, (uint32_t)((int64_t)M * a.Ci * 2));

  // This thread's copies: byte q*8192 + wave*1024 + lane*16 of the A and B
  // regions of a stage.  The row and the swizzled column it fills are the
  // same for every k tile; only the pixel advances.  A column outside the
  // operand gets a row index past any chunk, so its pixel test fails.
  constexpr int kDead = 1 << 30;
  int arow[SA], acol[SA];
#pragma unroll
  for (int q = 0; q < SA; ++q) {
    const int byte = q * NTHR * 16 + wave * 1024 + lane * 16;
    const int row = byte / ROWA;
    const int co = m0 + 8 * (((byte % ROWA) / 16) ^ swz(row));
    arow[q] = co < a.Co ? row : kDead;
    acol[q] = co;
  }
  int brow[SB], bci[SB], bdh[SB], bdw[SB];
#pragma unroll
  for (int q = 0; q < SB; ++q) {
    const int byte = q * NTHR * 16 + wave * 1024 + lane * 16;
    const int row = byte / ROWB;
    const int kk = n0 + 8 * (((byte % ROWB) / 16) ^ swz(row));
    brow[q] = kk < NW ? row : kDead;
    if constexpr (TAPS1) {
      bci[q] = kk; bdh[q] = 0; bdw[q] = 0;
    } else {
      const int rs = (int)fdiv((uint32_t)kk, fd_c);
      bci[q] = kk - rs * a.Ci;
      const int r = (rs * 11) >> 5;  // rs / 3 for rs < 9
      bdh[q] = r - 1;
      bdw[q] = rs - 3 * r - 1;
    }
  }

  // Tile kt >= nk starts at or past p_end: all its copies read zero.
  char *stage0 = smem + wave * 1024;
  auto issue = [&](int kt) {
    char *sa = stage0 + (kt % NS) * STAGE;
    const int pt = p_begin + kt * BK;
#pragma unroll
    for (int q = 0; q < SA; ++q) {
      const int p = pt + arow[q];
      const uint32_t off = p < p_end ? ((uint32_t)p * (uint32_t)a.Co + (uint32_t)acol[q]) * 2u : kOob;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsg, LDS_PTR(sa + q * NTHR * 16), 16, off, 0, 0, 0);
    }
#pragma unroll
    for (int q = 0; q < SB; ++q) {
      const int p = pt + brow[q];
      bool ok = p < p_end;
      int src = p;
      if constexpr (!TAPS1) {
        const uint32_t q1 = fdiv((uint32_t)p, fd_w);
        const int w = p - (int)q1 * a.W;
        const int h = (int)q1 - (int)fdiv(q1, fd_h) * a.H;
        ok = ok & ((unsigned)(h + bdh[q]) < (unsigned)a.H) & ((unsigned)(w + bdw[q]) < (unsigned)a.W);
        src = p + bdh[q] * a.W + bdw[q];
      }
      const uint32_t off = ok ? ((uint32_t)src * (uint32_t)a.Ci + (uint32_t)bci[q]) * 2u : kOob;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsx, LDS_PTR(sa + A_BYTES + q * NTHR * 16), 16, off, 0, 0, 0);
    }
  };

  // fragment read addresses (relative to a stage)
  const int j = lane & 15, lg = lane >> 4;
  const int wm = wave >> 2, wn = wave & 3;
  const int frow = 8 * lg + (j >> 2);
  const int fsw = swz(frow);
  const int half = ((j & 3) >> 1);
  uint32_t ra[4], rb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ra[i] = (uint32_t)(frow * ROWA + (((8 * wm + 2 * i + half) ^ fsw) * 16) + (j & 1) * 8);
    rb[i] = (uint32_t)(A_BYTES + frow * ROWB + (((8 * wn + 2 * i + half) ^ fsw) * 16) + (j & 1) * 8);
  }
  const uint32_t lds0 = (uint32_t)(size_t)LDS_PTR(smem);

  f32x4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[i][k] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  f32x4_t bacc = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Software pipeline over k tiles (R0/R1: fragments of k groups 0/1):
  //   wait R0; read R1; MFMA R0; wait R1       -- this tile's reads are done
  //   wait own copies of tile kt+1; barrier    -- kt+1 visible, stage kt free
  //   copy tile kt+3 into stage kt; read R0 of tile kt+1; MFMA R1
  // so the last MFMAs of a tile cover the next tile's first LDS reads.
  issue(0);
  issue(1);
  issue(2);
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * (SA + SB)) : "memory");
  asm volatile("s_barrier" ::: "memory");
  u32x4 a0[4], b0[4], a1[4], b1[4];
  if (nk > 0) read_group<0>(a0, b0, ra, rb, lds0);
  for (int kt = 0; kt < nk; ++kt) {
    const uint32_t st = lds0 + (uint32_t)((kt % NS) * STAGE);
    wait_lds(a0, b0);
    read_group<1>(a1, b1, ra, rb, st);
    mfma_group(acc, bacc, a0, b0, do_bias, wn);
    wait_lds(a1, b1);
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(SA + SB) : "memory");
    asm volatile("s_barrier" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    issue(kt + 3);
    if (kt + 1 < nk) read_group<0>(a0, b0, ra, rb, lds0 + (uint32_t)(((kt + 1) % NS) * STAGE));
    __builtin_amdgcn_sched_barrier(0);
    mfma_group(acc, bacc, a1, b1, do_bias, wn);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  float *dw = a.dw + split * a.dw_ss + rep * a.dw_rs;
#pragma unroll
  for (int tn = 0; tn < 4; ++tn) {
    const int n = n0 + wn * 64 + tn * 16 + j;
#pragma unroll
    for (int tm = 0; tm < 4; ++tm)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm * 64 + tm * 16 + lg * 4 + r;
        if (m < a.Co && n < a.nw) dw[(int64_t)m * a.nw + n] = acc[tm][tn][r];
      }
  }
  if (do_bias && j == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int co = m0 + wm * 64 + wn * 16 + lg * 4 + r;
      if (co < a.Co) a.db[split * a.db_ss + rep * a.db_rs + co] = bacc[r];
    }
  }
}

}  // namespace

bool wgrad_lds_ok(int dtype, int Co, int Ci) {
  return dtype == GCPSL_BF16 && Co >= 128 && Co % 8 == 0 && Ci % 8 == 0;
}

void wgrad_lds_tile(int *bm, int *bn, int *bk) {
  *bm = BM;
  *bn = BN;
  *bk = BK;
}

hipError_t launch_wgrad_lds(const WgradArgs &a, hipStream_t s, std::string *label) {
  static bool attr = false;
  if (!attr) {
    for (const void *f : {reinterpret_cast<const void *>(&wgrad_lds_kernel<true>),
                          reinterpret_cast<const void *>(&wgrad_lds_kernel<false>)}) {
      const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, LDS_BYTES);
      if (e != hipSuccess) return e;
    }
    attr = true;
  }
  const int NW = a.taps == 1 ? a.Ci : 9 * a.Ci;
  const int MT = (a.Co + BM - 1) / BM, NT = (NW + BN - 1) / BN;
  const FastDiv fw = make_fastdiv(a.W), fh = make_fastdiv(a.H), fc = make_fastdiv(a.Ci);
  const uint32_t blocks = (uint32_t)MT * NT * a.splits * a.C;
  if (label) *label = "conv_wgrad<bf16,128x256,w8,lds>";
  if (a.taps == 1)
    hipLaunchKernelGGL(wgrad_lds_kernel<true>, dim3(blocks), dim3(NTHR), LDS_BYTES, s, a, fw, fh, fc, MT, NT);
  else
    hipLaunchKernelGGL(wgrad_lds_kernel<false>, dim3(blocks), dim3(NTHR), LDS_BYTES, s, a, fw, fh, fc, MT, NT);
  return hipGetLastError();
}
