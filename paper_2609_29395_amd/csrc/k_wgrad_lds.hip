// Weight and bias gradient of a 3x3 conv layer, bf16, on gfx950:
//
//   dW[co][(r,s,ci)] = sum_p g[p][co] x[p + (r-1, s-1)][ci]      db[co] = sum_p g[p][co]
//
// with p = (b, h, w) running over a chunk of the batch's pixels (split-K).
// Both operands are stored pixel-major (NHWC): the reduction index is the
// outer dimension.  A k tile of 64 pixels is copied into LDS exactly as it
// lies in memory -- 64 rows of BM output channels (g) and 64 rows of BN
// im2col columns (x, shifted per kernel tap) -- by buffer loads that write LDS
// directly, so no registers stage the tiles and out-of-image taps,
// out-of-chunk pixels and ragged columns are zero-filled by the buffer range
// check.  The MFMA wants each lane to hold 8 consecutive k (pixels) of one
// output row or column; ds_read_b64_tr_b16 produces that from the
// pixel-major tile: within 16 lanes, lane 4r+q reads 4 channels of pixel r
// and lane i receives channel i of the 4 pixels.
//
// LDS rows are XOR-swizzled in 16-byte chunks (chunk ^ swz(row)) so that the
// 16 pixels of one transposing read fall on all banks.  The LDS reads are
// inline asm with explicit lgkmcnt waits so that the compiler does not add a
// wait for every outstanding copy before them.
//
// The workgroup tile is large (up to 256 x 256 outputs, 8 waves) because the
// per-CU vector-memory path bounds a k tile: the bytes copied per MFMA fall
// as the tile grows.  Two LDS stages: the copy of tile kt+1 is issued right
// after the barrier that starts tile kt and has all of tile kt's MFMAs to
// land.  The bias gradient rides along in the column-tile-0 workgroups: each
// wave multiplies BPW of its g fragments by a ones fragment (one extra MFMA
// per fragment and k group), together covering the workgroup's rows.
#include "runtime.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#define LDS_PTR(p) ((__attribute__((address_space(3))) void *)(p))

constexpr uint32_t kOob = 0x80000000u;
constexpr int kBufferFlags = 0x00020000;
constexpr int kDead = 1 << 30;  // row index that fails every pixel test

// BK pixels per k tile (a multiple of the 32 of one MFMA k group), NST LDS
// stages: the copies of a tile are issued NST - 1 tiles before it is used.
template <int BM, int BN, int WM, int WN, int BK_ = 64, int NST_ = 2> struct Cfg {
  static constexpr int BM_ = BM, BN_ = BN, WM_ = WM, WN_ = WN;
  static constexpr int BK = BK_, NST = NST_, KG = BK / 32;
  static constexpr int NW = WM * WN, NTHR = 64 * NW;  // waves, threads
  static constexpr int ROWA = BM * 2, ROWB = BN * 2;  // bytes per LDS row
  static constexpr int CHA = ROWA / 16, CHB = ROWB / 16;  // 16-byte chunks per row
  static constexpr int A_BYTES = BK * ROWA, B_BYTES = BK * ROWB;
  static constexpr int STAGE = A_BYTES + B_BYTES;
  static constexpr int SA = A_BYTES / (NTHR * 16), SB = B_BYTES / (NTHR * 16);  // copies per thread
  // rows between a thread's successive copies: a multiple of 16, so the
  // swizzled column (row bits 0, 1, 3) is the same for all of them
  static constexpr int QROWA = NTHR * 16 / ROWA, QROWB = NTHR * 16 / ROWB;
  static constexpr int TM = BM / WM / 16, TN = BN / WN / 16;                    // fragments per wave
  static constexpr int BPW = (TM + WN - 1) / WN;  // bias fragments per wave: those with tm % WN == wn
  static constexpr int LDS_BYTES = NST * STAGE;
  static constexpr int CPT = SA + SB;  // copies per thread per tile
  static constexpr int WNS = WN;
  static_assert(NW == 8 || NW == 16, "8 or 16 waves");
  static_assert(SA * NTHR * 16 == A_BYTES && SB * NTHR * 16 == B_BYTES, "copies must tile the stage");
  static_assert(QROWA % 16 == 0 && QROWB % 16 == 0, "copy rows keep the swizzle");
  static_assert(TM % WN == 0 || WN % TM == 0, "bias fragments split evenly over the waves of a row");
  static_assert(LDS_BYTES <= 160 * 1024, "LDS");
  static_assert(BK % 32 == 0 && NST >= 2, "k tile, stages");
};

// XOR applied to the 16-byte chunk index of LDS row `row` (CH chunks per
// row).  A transposing read touches 16 rows (4 per lane group, lane groups 8
// rows apart) at the same two chunks; the XOR spreads them so that each bank
// holds exactly two of the 16 pieces, and it depends only on row bits 0, 1
// and 3, which are the same for both halves of a fragment and for every k
// group.  Rows of 256 bytes or more start on bank 0; 128-byte rows alternate
// halves of the banks, so there the row's low bit already separates pairs.
template <int CH>
__device__ __forceinline__ int swz(int row) {
  static_assert(CH == 8 || CH >= 16, "row width");
  if constexpr (CH >= 16) return ((row & 3) | ((row >> 1) & 4)) << 1;
  else return (((row >> 1) & 1) | ((row >> 2) & 2)) << 1;
}

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

// Copies of k tile kt into its stage.  The buffer resources are built here
// from plain pointers: a buffer-resource value passed into a function or
// lambda of a kernel template makes the host compilation pass drop the
// kernel's launch stub without a diagnostic.
template <typename CF, bool TAPS1>
__device__ __forceinline__ void issue_tile(int kt, char *stage0, const WgradArgs &a, FastDiv fd_w, FastDiv fd_h,
                                           const void *G, const void *X, int M, int p_begin, int p_end,
                                           int arow, int acol, int brow, int bci, int btap) {
  const __amdgpu_buffer_rsrc_t rsg = rsrc(G, (uint32_t)((int64_t)M * a.Co * 2));
  const __amdgpu_buffer_rsrc_t rsx = rsrc(X, (uint32_t)((int64_t)M * a.Ci * 2));
  char *sa = stage0 + (kt % CF::NST) * CF::STAGE;
  const int pt = p_begin + kt * CF::BK;
#pragma unroll
  for (int q = 0; q < CF::SA; ++q) {
    const int p = pt + arow + q * CF::QROWA;
    const uint32_t off = p < p_end ? ((uint32_t)p * (uint32_t)a.Co + (uint32_t)acol) * 2u : kOob;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsg, LDS_PTR(sa + q * CF::NTHR * 16), 16, off, 0, 0, 0);
  }
#pragma unroll
  for (int q = 0; q < CF::SB; ++q) {
    const int p = pt + brow + q * CF::QROWB;
    bool ok = p < p_end;
    int src = p;
    if constexpr (!TAPS1) {
      const int dh = (btap & 3) - 1, dw = (btap >> 2) - 1;
      const uint32_t q1 = fdiv((uint32_t)p, fd_w);
      const int w = p - (int)q1 * a.W;
      const int h = (int)q1 - (int)fdiv(q1, fd_h) * a.H;
      ok = ok & ((unsigned)(h + dh) < (unsigned)a.H) & ((unsigned)(w + dw) < (unsigned)a.W);
      src = p + dh * a.W + dw;
    }
    const uint32_t off = ok ? ((uint32_t)src * (uint32_t)a.Ci + (uint32_t)bci) * 2u : kOob;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsx, LDS_PTR(sa + CF::A_BYTES + q * CF::NTHR * 16), 16, off, 0, 0, 0);
  }
}

// Fragments of k group KG (32 pixels) of the stage at byte address st, then
// their MFMAs; with bias, the g fragments tm with tm % WN == wn also meet a
// ones fragment (column sums of g).
template <typename CF, int KG>
__device__ __forceinline__ void kgroup(f32x4_t (&acc)[CF::TM][CF::TN], f32x4_t (&bacc)[CF::BPW],
                                       const uint32_t (&ra)[CF::TM], const uint32_t (&rb)[CF::TN], uint32_t st,
                                       bool bias, int wn) {
  constexpr int TM = CF::TM, TN = CF::TN;
  u32x4 a[TM], b[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) read_frag<KG * 32 * CF::ROWA, CF::ROWA>(a[i], st + ra[i]);
#pragma unroll
  for (int i = 0; i < TN; ++i) read_frag<KG * 32 * CF::ROWB, CF::ROWB>(b[i], st + rb[i]);
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int i = 0; i < TM; ++i) asm volatile("" : "+v"(a[i]));
#pragma unroll
  for (int i = 0; i < TN; ++i) asm volatile("" : "+v"(b[i]));
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) mma(acc[tm][tn], a[tm], b[tn]);
  if (bias) {
    const uint32_t one2 = 0x3F803F80u;  // two bf16 ones
    const u32x4 ones = u32x4{one2, one2, one2, one2};
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
      if (tm % CF::WNS == wn) mma(bacc[tm / CF::WNS], a[tm], ones);
  }
}

// s_waitcnt vmcnt(N) for a compile-time N
template <int N> __device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

template <int BM, int BN, int WM, int WN, int BK, int NST, bool TAPS1>
__global__ void __launch_bounds__(64 * WM * WN)
wgrad_lds_kernel(WgradArgs a, FastDiv fd_w, FastDiv fd_h, FastDiv fd_c, int MT, int NT) {
  using CF = Cfg<BM, BN, WM, WN, BK, NST>;
  constexpr int TM = CF::TM, TN = CF::TN, BPW = CF::BPW;
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
  const int rep = replica_of(a.rmap, __builtin_amdgcn_readfirstlane((int)(rest / (uint32_t)a.splits)));
  const int M = a.Bt * a.H * a.W;
  const int NW = a.taps == 1 ? a.Ci : 9 * a.Ci;
  const int p_begin = split * a.chunk;
  const int p_end = min(M, p_begin + a.chunk);
  const int nk = (p_end - p_begin + BK - 1) / BK;
  static_assert(CF::KG <= 2, "at most two k groups per tile");
  const int m0 = mt * BM, n0 = nt * BN;
  const bf16_t *G = reinterpret_cast<const bf16_t *>(a.g) + rep * a.g_rs;
  const bf16_t *X = reinterpret_cast<const bf16_t *>(a.x) + rep * a.x_rs;
  const bool do_bias = (nt == 0) && a.db != nullptr;

  // This thread's copies: bytes q*NTHR*16 + wave*1024 + lane*16 of the A and
  // B regions of a stage, i.e. rows row0 + q*QROW at one swizzled column.
  // Only the pixel advances from tile to tile.  A column outside the operand
  // gets a row index past any chunk, so its pixel test fails.
  const int byte0 = wave * 1024 + lane * 16;
  int arow, acol;
  {
    const int row = byte0 / CF::ROWA;
    acol = m0 + 8 * (((byte0 % CF::ROWA) / 16) ^ swz<CF::CHA>(row));
    arow = acol < a.Co ? row : kDead;
  }
  int brow, bci, btap;  // btap: (row offset + 1) | (column offset + 1) << 2
  {
    const int row = byte0 / CF::ROWB;
    const int kk = n0 + 8 * (((byte0 % CF::ROWB) / 16) ^ swz<CF::CHB>(row));
    brow = kk < NW ? row : kDead;
    if constexpr (TAPS1) {
      bci = kk; btap = 1 | (1 << 2);
    } else {
      const int rs = (int)fdiv((uint32_t)kk, fd_c);
      bci = kk - rs * a.Ci;
      const int r = (rs * 11) >> 5;  // rs / 3 for rs < 9
      btap = (r & 3) | (((rs - 3 * r) & 3) << 2);
    }
  }
  char *stage0 = smem + wave * 1024;

  // fragment read addresses (relative to a stage)
  const int j = lane & 15, lg = lane >> 4;
  const int wm = wave / WN, wn = wave % WN;
  const int frow = 8 * lg + (j >> 2);
  const int fsa = swz<CF::CHA>(frow), fsb = swz<CF::CHB>(frow);
  const int half = ((j & 3) >> 1);
  uint32_t ra[TM], rb[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
    ra[i] = (uint32_t)(frow * CF::ROWA + (((2 * (wm * TM + i) + half) ^ fsa) * 16) + (j & 1) * 8);
#pragma unroll
  for (int i = 0; i < TN; ++i)
    rb[i] = (uint32_t)(CF::A_BYTES + frow * CF::ROWB + (((2 * (wn * TN + i) + half) ^ fsb) * 16) + (j & 1) * 8);
  const uint32_t lds0 = (uint32_t)(size_t)LDS_PTR(smem);

  f32x4_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int k = 0; k < TN; ++k) acc[i][k] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  f32x4_t bacc[BPW];
#pragma unroll
  for (int i = 0; i < BPW; ++i) bacc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int q = 0; q < NST - 1; ++q)
    if (q < nk) issue_tile<CF, TAPS1>(q, stage0, a, fd_w, fd_h, G, X, M, p_begin, p_end, arow, acol, brow, bci, btap);
  for (int kt = 0; kt < nk; ++kt) {
    // own copies of tile kt have landed once only the copies of the tiles
    // issued after it (kt+1 .. kt+NST-2) are outstanding (vector memory
    // loads complete in order); near the end every copy is waited for.
    // After the barrier every wave's copies have landed and every wave is
    // done with tile kt-1, whose stage receives tile kt+NST-1.
    if (kt + NST - 2 < nk) wait_vm<(NST - 2) * CF::CPT>();
    else wait_vm<0>();
    asm volatile("s_barrier" ::: "memory");
    if (kt + NST - 1 < nk)
      issue_tile<CF, TAPS1>(kt + NST - 1, stage0, a, fd_w, fd_h, G, X, M, p_begin, p_end, arow, acol, brow, bci,
                            btap);
    const uint32_t st = lds0 + (uint32_t)((kt % NST) * CF::STAGE);
    kgroup<CF, 0>(acc, bacc, ra, rb, st, do_bias, wn);
    if constexpr (CF::KG > 1) kgroup<CF, 1>(acc, bacc, ra, rb, st, do_bias, wn);
  }
  // nk == 0 leaves the first copy in flight
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  float *dw = a.dw + split * a.dw_ss + rep * a.dw_rs;
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) {
    const int n = n0 + (wn * TN + tn) * 16 + j;
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + (wm * TM + tm) * 16 + lg * 4 + r;
        if (m < a.Co && n < a.nw) dw[(int64_t)m * a.nw + n] = acc[tm][tn][r];
      }
  }
  if (do_bias && j == 0) {
#pragma unroll
    for (int i = 0; i < BPW; ++i) {
      const int tm = wn + WN * i;
      if (tm >= TM) break;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int co = m0 + (wm * TM + tm) * 16 + lg * 4 + r;
        if (co < a.Co) a.db[split * a.db_ss + rep * a.db_rs + co] = bacc[i][r];
      }
    }
  }
}

// ------------------------------------------------------------- halo mode
// 16 x 16 images, output channels a multiple of 128, input channels a
// multiple of 64 (the wide server layers).  A workgroup owns 128 output
// channels x one 64-channel input block x all nine taps (128 x 576 outputs).
// A k tile of 128 pixels is eight image rows (half an image); what every tap
// needs of the input is the ten image rows around them with a one-pixel
// zero border, 10 x 18 pixel rows of 128 bytes, copied once; the nine taps
// read their fragments from it at shifted rows.  A k tile then copies 32 KB
// of g and 22.5 KB of input for 18.9 MFLOP, against 128 KB for 16.8 MFLOP
// with one tap per 256 x 256 tile; four k groups of two image rows share one
// barrier.
// Halo row R = 18 h' + w' stores its 16-byte chunk c at c ^ 2 whsw(w'),
// whsw(w') = bit 1 of w' | (bit 3 of w') << 1: the eight rows a half-wave's
// transposing read touches (w' in {a .. a+3, a+8 .. a+11} for one image row)
// then use every bank exactly once, and the rows of successive image rows and
// of the three kernel-tap rows sit a constant 18 rows (2,304 bytes) apart.
namespace wh {
constexpr int IMG = 16, HP = 18, TR = 8;   // image side, halo row width, image rows per k tile
constexpr int BK = IMG * TR;               // 128 pixels per k tile
constexpr int HROWS = (TR + 2) * HP;       // 180 halo rows
constexpr int ROWB = 128;                  // bytes per halo row (64 channels)
constexpr int BM = 128, ROWA = BM * 2;     // output channels per workgroup, bytes per g row
constexpr int NTHR = 512, TM = 4;          // 8 waves (2 x 4); g fragments per wave
constexpr int A_BYTES = BK * ROWA;         // 32 KB
constexpr int B_BYTES = 24576;             // 180 halo rows, the rest takes the zero copies of idle lanes
constexpr int STAGE = A_BYTES + B_BYTES;
constexpr int SA = A_BYTES / (NTHR * 16), SB = B_BYTES / (NTHR * 16), CPT = SA + SB;
constexpr int QROWA = NTHR * 16 / ROWA;    // g rows between a thread's copies
constexpr int FROW = HP * ROWB;            // bytes between halo image rows
static_assert(HROWS * ROWB <= B_BYTES && SA == 4 && SB == 3 && QROWA % 16 == 0, "halo weight-gradient layout");
}  // namespace wh
__device__ __forceinline__ int whsw(int wp) { return ((wp >> 1) & 1) | ((wp >> 2) & 2); }

// One operand fragment from two transposing reads at separate addresses (the
// halo's swizzle differs between the two 4-pixel halves).
template <int OFF>
__device__ __forceinline__ void read_frag2(u32x4 &f, uint32_t a0, uint32_t a1) {
  u32x2 lo, hi;
  asm volatile("ds_read_b64_tr_b16 %0, %2 offset:%4\n\tds_read_b64_tr_b16 %1, %3 offset:%4"
               : "=&v"(lo), "=&v"(hi)
               : "v"(a0), "v"(a1), "n"(OFF));
  f = __builtin_shufflevector(lo, hi, 0, 1, 2, 3);
}

// Copies of k tile kt into stage kt % NST: g rows (pixels) at this thread's
// column, and this thread's halo rows (hh = h' of the row, -1 for the zero
// border and padding; hrel = its source offset from the tile's first pixel).
template <int NST>
__device__ __forceinline__ void wh_issue(int kt, char *stage0, const void *G, const void *X, uint32_t gbytes,
                                         uint32_t xbytes, int Co, int Ci, int p_begin, int arow, int acol,
                                         const int (&hrel)[wh::SB], const int (&hh)[wh::SB]) {
  const __amdgpu_buffer_rsrc_t rsg = rsrc(G, gbytes);
  const __amdgpu_buffer_rsrc_t rsx = rsrc(X, xbytes);
  char *sa = stage0 + (kt % NST) * wh::STAGE;
  const int pt = p_begin + kt * wh::BK;
#pragma unroll
  for (int q = 0; q < wh::SA; ++q) {
    const uint32_t off = ((uint32_t)(pt + arow + q * wh::QROWA) * (uint32_t)Co + (uint32_t)acol) * 2u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsg, LDS_PTR(sa + q * wh::NTHR * 16), 16, off, 0, 0, 0);
  }
  const int h0 = (pt >> 4) & (wh::IMG - 1);  // first image row of the tile
#pragma unroll
  for (int q = 0; q < wh::SB; ++q) {
    const bool ok = hh[q] >= 0 && (unsigned)(h0 - 1 + hh[q]) < (unsigned)wh::IMG;
    const uint32_t off = ok ? (uint32_t)(pt * Ci + hrel[q]) * 2u : kOob;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsx, LDS_PTR(sa + wh::A_BYTES + q * wh::NTHR * 16), 16, off, 0, 0, 0);
  }
}

// k group KG (image rows 2 KG, 2 KG + 1) of the stage at st: 4 g fragments, one input
// fragment per tap, 36 MFMAs (+1 against ones for the bias gradient).
template <int KG>
__device__ __forceinline__ void wh_kgroup(f32x4_t (&acc)[wh::TM][9], f32x4_t &bacc, const uint32_t (&ra)[wh::TM],
                                          const uint32_t (&hb)[3][2], uint32_t st, bool bias, int wn) {
  u32x4 a[wh::TM], b[9];
#pragma unroll
  for (int i = 0; i < wh::TM; ++i) read_frag<KG * 32 * wh::ROWA, wh::ROWA>(a[i], st + ra[i]);
  constexpr int O = wh::A_BYTES + KG * 2 * wh::FROW;
  read_frag2<O + 0 * wh::FROW>(b[0], st + hb[0][0], st + hb[0][1]);
  read_frag2<O + 0 * wh::FROW>(b[1], st + hb[1][0], st + hb[1][1]);
  read_frag2<O + 0 * wh::FROW>(b[2], st + hb[2][0], st + hb[2][1]);
  read_frag2<O + 1 * wh::FROW>(b[3], st + hb[0][0], st + hb[0][1]);
  read_frag2<O + 1 * wh::FROW>(b[4], st + hb[1][0], st + hb[1][1]);
  read_frag2<O + 1 * wh::FROW>(b[5], st + hb[2][0], st + hb[2][1]);
  read_frag2<O + 2 * wh::FROW>(b[6], st + hb[0][0], st + hb[0][1]);
  read_frag2<O + 2 * wh::FROW>(b[7], st + hb[1][0], st + hb[1][1]);
  read_frag2<O + 2 * wh::FROW>(b[8], st + hb[2][0], st + hb[2][1]);
  // LDS reads complete in order: the g fragments and tap row 0 are in after
  // all but the last 12 of the 26 reads, tap row 1 after all but 6
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_waitcnt lgkmcnt(12)" ::: "memory");
#pragma unroll
  for (int i = 0; i < wh::TM; ++i) asm volatile("" : "+v"(a[i]));
#pragma unroll
  for (int i = 0; i < 3; ++i) asm volatile("" : "+v"(b[i]));
#pragma unroll
  for (int tm = 0; tm < wh::TM; ++tm)
#pragma unroll
    for (int tap = 0; tap < 3; ++tap) mma(acc[tm][tap], a[tm], b[tap]);
  __builtin_amdgcn_sched_barrier(0);  // keep these MFMAs ahead of the next wait
  asm volatile("s_waitcnt lgkmcnt(6)" ::: "memory");
#pragma unroll
  for (int i = 3; i < 6; ++i) asm volatile("" : "+v"(b[i]));
#pragma unroll
  for (int tm = 0; tm < wh::TM; ++tm)
#pragma unroll
    for (int tap = 3; tap < 6; ++tap) mma(acc[tm][tap], a[tm], b[tap]);
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int i = 6; i < 9; ++i) asm volatile("" : "+v"(b[i]));
#pragma unroll
  for (int tm = 0; tm < wh::TM; ++tm)
#pragma unroll
    for (int tap = 6; tap < 9; ++tap) mma(acc[tm][tap], a[tm], b[tap]);
  if (bias) {
    const uint32_t one2 = 0x3F803F80u;  // two bf16 ones
    const u32x4 ones = u32x4{one2, one2, one2, one2};
#pragma unroll
    for (int tm = 0; tm < wh::TM; ++tm)
      if (tm == wn) mma(bacc, a[tm], ones);
  }
}

template <int NST>
__global__ void __launch_bounds__(wh::NTHR)
wgrad_halo_kernel(WgradArgs a, int MT, int NT) {
  constexpr int TM = wh::TM;
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t total = (uint32_t)(MT * NT * a.splits * a.C);
  const uint32_t t = xcd_swizzle(blockIdx.x, total);
  const int cb = __builtin_amdgcn_readfirstlane((int)(t % (uint32_t)NT));  // input-channel block
  uint32_t rest = t / (uint32_t)NT;
  const int mt = __builtin_amdgcn_readfirstlane((int)(rest % (uint32_t)MT));
  rest /= (uint32_t)MT;
  const int split = __builtin_amdgcn_readfirstlane((int)(rest % (uint32_t)a.splits));
  const int rep = replica_of(a.rmap, __builtin_amdgcn_readfirstlane((int)(rest / (uint32_t)a.splits)));
  const int M = a.Bt * wh::IMG * wh::IMG;
  const int p_begin = split * a.chunk;
  const int p_end = min(M, p_begin + a.chunk);
  const int nk = (p_end - p_begin) / wh::BK;
  const int m0 = mt * wh::BM;
  const bf16_t *G = reinterpret_cast<const bf16_t *>(a.g) + rep * a.g_rs;
  const bf16_t *X = reinterpret_cast<const bf16_t *>(a.x) + rep * a.x_rs;
  const uint32_t gbytes = (uint32_t)((int64_t)M * a.Co * 2), xbytes = (uint32_t)((int64_t)M * a.Ci * 2);
  const bool do_bias = (cb == 0) && a.db != nullptr;

  // this thread's copies: bytes q*8192 + wave*1024 + lane*16 of each region
  const int byte0 = wave * 1024 + lane * 16;
  const int arow = byte0 / wh::ROWA;
  const int acol = m0 + 8 * (((byte0 % wh::ROWA) / 16) ^ swz<wh::ROWA / 16>(arow));
  int hrel[wh::SB], hh[wh::SB];
#pragma unroll
  for (int q = 0; q < wh::SB; ++q) {
    const int R = (q * wh::NTHR * 16 + byte0) / wh::ROWB, cs = (byte0 / 16) & 7;
    const int hp = R / wh::HP, wp = R - wh::HP * hp;
    const int c = cs ^ (2 * whsw(wp));
    const bool in = R < wh::HROWS && wp >= 1 && wp <= wh::IMG;
    hh[q] = in ? hp : -1;
    hrel[q] = ((hp - 1) * wh::IMG + (wp - 1)) * a.Ci + cb * 64 + 8 * c;
  }
  char *stage0 = smem + wave * 1024;

  // fragment read addresses (relative to a stage)
  const int j = lane & 15, lg = lane >> 4;
  const int wm = wave >> 2, wn = wave & 3;
  const int frow = 8 * lg + (j >> 2);
  const int half = (j & 3) >> 1;
  uint32_t ra[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i)
    ra[i] = (uint32_t)(frow * wh::ROWA + (((2 * (wm * TM + i) + half) ^ swz<wh::ROWA / 16>(frow)) * 16) + (j & 1) * 8);
  // input fragments of tap column s, halves rd: pixel 8 lg + 4 rd + j / 4 of
  // the k group is image row lg / 2, column 8 (lg & 1) + 4 rd + j / 4
  uint32_t hb[3][2];
#pragma unroll
  for (int s = 0; s < 3; ++s)
#pragma unroll
    for (int rd = 0; rd < 2; ++rd) {
      const int wp = (lg & 1) * 8 + 4 * rd + (j >> 2) + s;
      const int R = (lg >> 1) * wh::HP + wp;
      hb[s][rd] = (uint32_t)(R * wh::ROWB + (((2 * wn + half) ^ (2 * whsw(wp))) * 16) + (j & 1) * 8);
    }
  const uint32_t lds0 = (uint32_t)(size_t)LDS_PTR(smem);

  f32x4_t acc[TM][9];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int k = 0; k < 9; ++k) acc[i][k] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  f32x4_t bacc = f32x4_t{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int q = 0; q < NST - 1; ++q)
    if (q < nk)
      wh_issue<NST>(q, stage0, G, X, gbytes, xbytes, a.Co, a.Ci, p_begin, arow, acol, hrel, hh);
  for (int kt = 0; kt < nk; ++kt) {
    // as in the generic kernel: own copies of tile kt have landed once only
    // those of tiles kt+1 .. kt+NST-2 are outstanding; after the barrier all
    // waves' copies have landed and tile kt-1's stage is free
    if (kt + NST - 2 < nk) wait_vm<(NST - 2) * wh::CPT>();
    else wait_vm<0>();
    asm volatile("s_barrier" ::: "memory");
    if (kt + NST - 1 < nk)
      wh_issue<NST>(kt + NST - 1, stage0, G, X, gbytes, xbytes, a.Co, a.Ci, p_begin, arow, acol, hrel, hh);
    const uint32_t st = lds0 + (uint32_t)((kt % NST) * wh::STAGE);
    wh_kgroup<0>(acc, bacc, ra, hb, st, do_bias, wn);
    wh_kgroup<1>(acc, bacc, ra, hb, st, do_bias, wn);
    wh_kgroup<2>(acc, bacc, ra, hb, st, do_bias, wn);
    wh_kgroup<3>(acc, bacc, ra, hb, st, do_bias, wn);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  float *dw = a.dw + split * a.dw_ss + rep * a.dw_rs;
#pragma unroll
  for (int tap = 0; tap < 9; ++tap) {
    const int n = tap * a.Ci + cb * 64 + wn * 16 + j;
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + (wm * TM + tm) * 16 + lg * 4 + r;
        dw[(int64_t)m * a.nw + n] = acc[tm][tap][r];
      }
  }
  if (do_bias && j == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int co = m0 + (wm * TM + wn) * 16 + lg * 4 + r;
      a.db[split * a.db_ss + rep * a.db_rs + co] = bacc[r];
    }
  }
}

// ------------------------------------------------- image-side client layer
// 32 x 32 images, 64 output and 32 input channels (the layer between the
// image layer and the cut).  A workgroup owns the whole 64 x 288 gradient
// (nine taps x 32 input channels) for its pixel chunk: 8 waves, wave (wm, wn)
// takes output channels 16 wm .. 16 wm + 15 and column fragments 9 wn ..
// 9 wn + 8 (fragment f = tap * 2 + 16-channel block), 36 accumulator registers
// per lane.  A k tile is 64 pixels = two image rows; the input rows all taps
// need (four image rows with a zero border, 4 x 34 pixel rows of 64 bytes)
// are copied once, next to the 64 x 64 g tile.  Halo row R (column w') keeps
// its 16-byte chunk c at c ^ wisw(w').
namespace wi {
constexpr int IMG = 32, HP = 34, TR = 2;    // image side, halo row width, image rows per k tile
constexpr int BK = IMG * TR;                // 64 pixels per k tile
constexpr int HROWS = (TR + 2) * HP;        // 136 halo rows
constexpr int CI = 32, CO = 64;             // input and output channels
constexpr int ROWB = CI * 2;                // 64 bytes per halo row
constexpr int ROWA = CO * 2;                // 128 bytes per g row
constexpr int NTHR = 512;
constexpr int A_BYTES = BK * ROWA;          // 8 KB
constexpr int B_BYTES = 16384;              // 136 halo rows (8.5 KB); the rest takes idle lanes' zero copies
constexpr int STAGE = A_BYTES + B_BYTES;
constexpr int SA = A_BYTES / (NTHR * 16), SB = B_BYTES / (NTHR * 16), CPT = SA + SB;
constexpr int QROWA = NTHR * 16 / ROWA;     // g rows between a thread's copies
constexpr int FROW = HP * ROWB;             // bytes between halo image rows
constexpr int NF = 9;                       // column fragments per wave
// routed g tile (POOL): the pooled gradient row and its codes in the B
// region's tail, after the halo rows and 32 zero pieces
constexpr int PROW_G = (IMG / 2) * CO * 2;  // 2 KB: one pooled row of gradient
constexpr int PROW_C = (IMG / 2) * CO;      // 1 KB: its codes
constexpr int RAW_G = NTHR * 16 + 1024, RAW_C = RAW_G + PROW_G, IDLE = RAW_C + PROW_C;
static_assert(HROWS * ROWB <= B_BYTES && SA == 1 && SB == 2 && QROWA % 16 == 0, "image weight-gradient layout");
static_assert(HROWS * ROWB <= RAW_G && IDLE + 4 * 1024 <= B_BYTES && PROW_G == 2048 && PROW_C == 1024,
              "routed g tile in the B region's tail");
}  // namespace wi
__device__ __forceinline__ int wisw(int wp) { return (wp >> 1) & 3; }

// Copies of k tile kt into stage kt % NST.  Plain: the g tile (A region)
// and the input halo rows (B region, two copies per thread).  POOL: the g
// tile is routed in LDS (wi_route) from the pooled gradient and its codes,
// which the second copy brings into the B region's idle tail: waves 0 and 1
// the tile's pooled gradient row (2 KB at RAW_G), wave 2 its codes (1 KB at
// RAW_C), wave 7 the last 32 halo pieces (and 32 zero pieces after them),
// waves 3 .. 6 zero copies into the rest of the tail.  Each copy instruction
// stays with one source buffer per wave.  The second copy is issued first,
// so that the routed tile can be waited for ahead of the halo copies.
template <int NST, bool POOL>
__device__ __forceinline__ void wi_issue(int kt, char *smem, int wave, int lane, const void *G, const void *X,
                                         const void *code, uint32_t gbytes, uint32_t xbytes, int p_begin, int arow,
                                         int acol, const int (&hrel)[wi::SB], const int (&hh)[wi::SB]) {
  const __amdgpu_buffer_rsrc_t rsg = rsrc(G, gbytes);
  const __amdgpu_buffer_rsrc_t rsx = rsrc(X, xbytes);
  char *st = smem + (kt % NST) * wi::STAGE;
  const int pt = p_begin + kt * wi::BK;
  const int h0 = (pt / wi::IMG) % wi::IMG;  // first image row of the tile
  auto halo_off = [&](int q) {
    const bool ok = hh[q] >= 0 && (unsigned)(h0 - 1 + hh[q]) < (unsigned)wi::IMG;
    return ok ? (uint32_t)(pt * wi::CI + hrel[q]) * 2u : kOob;
  };
  if constexpr (!POOL) {
#pragma unroll
    for (int q = 0; q < wi::SA; ++q) {
      const uint32_t off = ((uint32_t)(pt + arow + q * wi::QROWA) * (uint32_t)wi::CO + (uint32_t)acol) * 2u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsg, LDS_PTR(st + wave * 1024 + q * wi::NTHR * 16), 16, off, 0, 0, 0);
    }
#pragma unroll
    for (int q = 0; q < wi::SB; ++q)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsx, LDS_PTR(st + wi::A_BYTES + wave * 1024 + q * wi::NTHR * 16), 16,
                                               halo_off(q), 0, 0, 0);
  } else {
    static_assert(wi::SB == 2 && wi::NTHR == 512 && wi::HROWS * wi::ROWB == wi::NTHR * 16 + 32 * 16,
                  "the second copy holds 32 halo pieces");
    const int prow = pt / wi::BK;  // pooled row of the replica (a tile is two image rows)
    char *sb = st + wi::A_BYTES;
    // (offsets from an opaque copy of the thread index, recomputed at each
    // issue rather than held in registers across the k loop)
    int t16 = (int)threadIdx.x * 16;
    asm volatile("" : "+v"(t16));
    if (wave == 7) {
      // halo pieces 512 + lane = halo rows 128 + lane / 4: halo image row 3
      // (image row h0 + 2), columns 26 + lane / 4, inside the image for
      // lanes 0 .. 27; the rest are the right border and zero pieces
      static_assert(wi::NTHR * 16 / wi::ROWB == 3 * wi::HP + 26 && wi::HROWS == 4 * wi::HP, "halo tail");
      const int ln = (t16 >> 4) & 63, wp = 26 + (ln >> 2), c = (ln & 3) ^ wisw(wp);
      const bool ok = ln < 28 && (unsigned)(h0 + 2) < (unsigned)wi::IMG;
      const uint32_t off = ok ? (uint32_t)(pt * wi::CI + (2 * wi::IMG + wp - 1) * wi::CI + 8 * c) * 2u : kOob;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsx, LDS_PTR(sb + wi::NTHR * 16), 16, off, 0, 0, 0);
    } else if (wave < 2) {
      const uint32_t off = (uint32_t)(prow * wi::PROW_G + t16);  // wave * 1024 + lane * 16
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsg, LDS_PTR(sb + wi::RAW_G + wave * 1024), 16, off, 0, 0, 0);
    } else if (wave == 2) {
      const __amdgpu_buffer_rsrc_t rsc = rsrc(code, gbytes / 2);
      const uint32_t off = (uint32_t)(prow * wi::PROW_C + t16 - 2048);  // lane * 16
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsc, LDS_PTR(sb + wi::RAW_C), 16, off, 0, 0, 0);
    } else {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsx, LDS_PTR(sb + wi::IDLE + (wave - 3) * 1024), 16, kOob, 0, 0, 0);
    }
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsx, LDS_PTR(sb + wave * 1024), 16, halo_off(0), 0, 0, 0);
  }
}

// POOL: this thread's piece of the g tile in the stage (pixel row arow,
// channels acol .. acol + 7, at byte 16 tid as a copy would put it) is the
// pooled gradient of its 2 x 2 window where the window's routing code names
// the pixel's position, zero elsewhere.  A tile is two image rows from an
// even row, so the pixel's window is pooled column (arow mod 32) / 2 of the
// tile's pooled row and its position is fixed by arow.
__device__ __forceinline__ void wi_route(char *st, int tid, int arow, int acol) {
  const int pc = (arow % wi::IMG) >> 1;
  const uint32_t pos = (uint32_t)((((arow / wi::IMG) & 1) << 1) | (arow & 1));
  const u32x4 g = *reinterpret_cast<const u32x4 *>(st + wi::A_BYTES + wi::RAW_G + pc * wi::ROWA + acol * 2);
  const u32x2 code = *reinterpret_cast<const u32x2 *>(st + wi::A_BYTES + wi::RAW_C + pc * wi::CO + acol);
  u32x4 v;
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const uint32_t cb = code[d >> 1] >> (16 * (d & 1));  // codes of channels 2d, 2d + 1
    const uint32_t keep = ((cb & 0xffu) == pos ? 0x0000ffffu : 0u) | (((cb >> 8) & 0xffu) == pos ? 0xffff0000u : 0u);
    v[d] = g[d] & keep;
  }
  *reinterpret_cast<u32x4 *>(st + tid * 16) = v;
}

// k group KG (image row KG of the tile): one g fragment, nine input
// fragments, nine MFMAs (+1 against ones for the bias gradient).
template <int KG>
__device__ __forceinline__ void wi_kgroup(f32x4_t (&acc)[wi::NF], f32x4_t &bacc, uint32_t ra,
                                          const uint32_t (&hb)[3][2][2], uint32_t st, bool bias, int wn) {
  u32x4 a, b[wi::NF];
  read_frag<KG * 32 * wi::ROWA, wi::ROWA>(a, st + ra);
  // fragment f = 9 wn + i: tap t = f / 2 (r = t / 3, s = t % 3), block f % 2
#pragma unroll
  for (int i = 0; i < wi::NF; ++i) {
    const int f0 = i, f1 = 9 + i;  // the wave's fragment for wn = 0 / 1
    const int t0 = f0 / 2, t1 = f1 / 2;
    // both choices are compile-time constants; wn selects one at run time
    const uint32_t s0 = st + hb[t0 % 3][f0 % 2][0], s1 = st + hb[t1 % 3][f1 % 2][0];
    const uint32_t e0 = st + hb[t0 % 3][f0 % 2][1], e1 = st + hb[t1 % 3][f1 % 2][1];
    const uint32_t lo = wn ? s1 : s0, hi = wn ? e1 : e0;
    const int r = wn ? t1 / 3 : t0 / 3;
    const uint32_t ro = (uint32_t)(r * wi::FROW);
    u32x2 l2, h2;
    asm volatile("ds_read_b64_tr_b16 %0, %2 offset:%4\n\tds_read_b64_tr_b16 %1, %3 offset:%4"
                 : "=&v"(l2), "=&v"(h2)
                 : "v"(lo + ro), "v"(hi + ro), "n"(wi::A_BYTES + KG * wi::FROW));
    b[i] = __builtin_shufflevector(l2, h2, 0, 1, 2, 3);
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  asm volatile("" : "+v"(a));
#pragma unroll
  for (int i = 0; i < wi::NF; ++i) asm volatile("" : "+v"(b[i]));
#pragma unroll
  for (int i = 0; i < wi::NF; ++i) mma(acc[i], a, b[i]);
  if (bias) {
    const uint32_t one2 = 0x3F803F80u;  // two bf16 ones
    mma(bacc, a, u32x4{one2, one2, one2, one2});
  }
}

// one k group (image row kw of the tile: its g rows from sa, its input rows
// from st) for 32 output channels: two g fragments (the second's chunk
// differs from the first's in bit 1 of the swizzled chunk index: address
// bit 5) and the wave's nine input fragments, read two at a time; eighteen
// MFMAs (+2 against ones for the bias gradient)
template <int I0, int NB>
__device__ __forceinline__ void wi_bfrags(u32x4 (&b)[2], const uint32_t (&hb)[3][2][2], uint32_t st, int wn) {
#pragma unroll
  for (int u = 0; u < NB; ++u) {
    // fragment f = 9 wn + i: tap t = f / 2 (r = t / 3, s = t % 3), block f % 2
    const int i = I0 + u;
    const int f0 = i, f1 = 9 + i;  // the wave's fragment for wn = 0 / 1
    const int t0 = f0 / 2, t1 = f1 / 2;
    // both choices are compile-time constants; wn selects one at run time
    const uint32_t s0 = st + hb[t0 % 3][f0 % 2][0], s1 = st + hb[t1 % 3][f1 % 2][0];
    const uint32_t e0 = st + hb[t0 % 3][f0 % 2][1], e1 = st + hb[t1 % 3][f1 % 2][1];
    const uint32_t lo = wn ? s1 : s0, hi = wn ? e1 : e0;
    const int r = wn ? t1 / 3 : t0 / 3;
    const uint32_t ro = (uint32_t)(r * wi::FROW);
    u32x2 l2, h2;
    asm volatile("ds_read_b64_tr_b16 %0, %2 offset:%4\n\tds_read_b64_tr_b16 %1, %3 offset:%4"
                 : "=&v"(l2), "=&v"(h2)
                 : "v"(lo + ro), "v"(hi + ro), "n"(wi::A_BYTES));
    b[u] = __builtin_shufflevector(l2, h2, 0, 1, 2, 3);
  }
}

__device__ __forceinline__ void wi_kgroup2(f32x4_t (&acc)[2][wi::NF], f32x4_t (&bacc)[2], uint32_t ra,
                                           const uint32_t (&hb)[3][2][2], uint32_t sa, uint32_t st, bool bias,
                                           int wn) {
  u32x4 a[2];
  read_frag<0, wi::ROWA>(a[0], sa + ra);
  read_frag<0, wi::ROWA>(a[1], sa + (ra ^ 32u));
  auto step = [&](const u32x4 (&b)[2], int i0, int nb) {
#pragma unroll
    for (int u = 0; u < 2; ++u)
      if (u < nb) {
        mma(acc[0][i0 + u], a[0], b[u]);
        mma(acc[1][i0 + u], a[1], b[u]);
      }
  };
  u32x4 b[2];
#define WI_GROUP(I0, NB)                                   \
  wi_bfrags<I0, NB>(b, hb, st, wn);                        \
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");       \
  asm volatile("" : "+v"(a[0]), "+v"(a[1]));               \
  asm volatile("" : "+v"(b[0]), "+v"(b[1]));               \
  step(b, I0, NB);
  WI_GROUP(0, 2)
  WI_GROUP(2, 2)
  WI_GROUP(4, 2)
  WI_GROUP(6, 2)
  WI_GROUP(8, 1)
#undef WI_GROUP
  if (bias) {
    const uint32_t one2 = 0x3F803F80u;  // two bf16 ones
    mma(bacc[0], a[0], u32x4{one2, one2, one2, one2});
    mma(bacc[1], a[1], u32x4{one2, one2, one2, one2});
  }
}

// (at least four waves per SIMD: at most 128 registers, so that two
// workgroups share a CU)
template <int NST, bool POOL>
__global__ void __launch_bounds__(wi::NTHR, 4)
wgrad_img_kernel(WgradArgs a) {
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t total = (uint32_t)(a.splits * a.C);
  const uint32_t t = xcd_swizzle(blockIdx.x, total);
  const int split = __builtin_amdgcn_readfirstlane((int)(t % (uint32_t)a.splits));
  const int rep = replica_of(a.rmap, __builtin_amdgcn_readfirstlane((int)(t / (uint32_t)a.splits)));
  const int M = a.Bt * wi::IMG * wi::IMG;
  const int p_begin = split * a.chunk;
  const int p_end = min(M, p_begin + a.chunk);
  const int nk = (p_end - p_begin) / wi::BK;
  const bf16_t *G = reinterpret_cast<const bf16_t *>(a.g) + rep * a.g_rs;
  const bf16_t *X = reinterpret_cast<const bf16_t *>(a.x) + rep * a.x_rs;
  const uint8_t *gc = POOL ? a.gcode + rep * a.g_rs : nullptr;
  // (POOL: g and gc are the pooled gradient and its codes, a quarter of the pixels)
  const uint32_t gbytes = (uint32_t)((int64_t)M * wi::CO * 2 / (POOL ? 4 : 1)),
                 xbytes = (uint32_t)((int64_t)M * wi::CI * 2);
  // wave (kw, wm2, wn): image row kw of every k tile, output channels
  // 32 wm2 .. + 31, input fragments 9 wn .. 9 wn + 8; the two k rows' sums
  // are added at the end
  const int kw = wave >> 2, wm2 = (wave >> 1) & 1, wn = wave & 1;
  const bool do_bias = wn == 0 && a.db != nullptr;

  // this thread's copies: bytes q*8192 + wave*1024 + lane*16 of each region
  const int byte0 = wave * 1024 + lane * 16;
  const int arow = byte0 / wi::ROWA;
  const int acol = 8 * (((byte0 % wi::ROWA) / 16) ^ swz<wi::ROWA / 16>(arow));
  int hrel[wi::SB], hh[wi::SB];
#pragma unroll
  for (int q = 0; q < wi::SB; ++q) {  // (POOL: piece 0 only)
    const int b0 = byte0;
    const int R = (q * wi::NTHR * 16 + b0) / wi::ROWB, cs = (b0 / 16) & 3;
    const int hp = R / wi::HP, wp = R - wi::HP * hp;
    const int c = cs ^ wisw(wp);
    const bool in = R < wi::HROWS && wp >= 1 && wp <= wi::IMG;
    hh[q] = in ? hp : -1;
    hrel[q] = ((hp - 1) * wi::IMG + (wp - 1)) * wi::CI + 8 * c;
  }

  // fragment read addresses (relative to a stage): g fragment of output
  // channels 16 wm.., input fragment halves of tap column s, channel block cb
  const int j = lane & 15, lg = lane >> 4;
  const int frow = 8 * lg + (j >> 2);
  const int half = (j & 3) >> 1;
  const uint32_t ra =
      (uint32_t)(frow * wi::ROWA + (((4 * wm2 + half) ^ swz<wi::ROWA / 16>(frow)) * 16) + (j & 1) * 8);
  static_assert(wi::ROWA == 128, "g fragment chunk index in address bits 4..6");
  uint32_t hb[3][2][2];
#pragma unroll
  for (int s = 0; s < 3; ++s)
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
      for (int rd = 0; rd < 2; ++rd) {
        const int wp = 8 * lg + 4 * rd + (j >> 2) + s;
        hb[s][cb][rd] = (uint32_t)(wp * wi::ROWB + (((2 * cb + half) ^ wisw(wp)) * 16) + (j & 1) * 8);
      }
  const uint32_t lds0 = (uint32_t)(size_t)LDS_PTR(smem);

  f32x4_t acc[2][wi::NF];
#pragma unroll
  for (int r2 = 0; r2 < 2; ++r2)
#pragma unroll
    for (int i = 0; i < wi::NF; ++i) acc[r2][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  f32x4_t bacc[2] = {f32x4_t{0.f, 0.f, 0.f, 0.f}, f32x4_t{0.f, 0.f, 0.f, 0.f}};
  // (the wave's k row: 32 g rows and one halo image row further)
  const uint32_t koa = (uint32_t)(kw * 32 * wi::ROWA), kob = (uint32_t)(kw * wi::FROW);
  auto kgroups = [&](uint32_t st) { wi_kgroup2(acc, bacc, ra, hb, st + koa, st + kob, do_bias, wn); };

  if constexpr (!POOL) {
#pragma unroll
    for (int q = 0; q < NST - 1; ++q)
      if (q < nk) wi_issue<NST, false>(q, smem, wave, lane, G, X, gc, gbytes, xbytes, p_begin, arow, acol, hrel, hh);
    for (int kt = 0; kt < nk; ++kt) {
      if (kt + NST - 2 < nk) wait_vm<(NST - 2) * wi::CPT>();
      else wait_vm<0>();
      asm volatile("s_barrier" ::: "memory");
      if (kt + NST - 1 < nk)
        wi_issue<NST, false>(kt + NST - 1, smem, wave, lane, G, X, gc, gbytes, xbytes, p_begin, arow, acol, hrel, hh);
      kgroups(lds0 + (uint32_t)((kt % NST) * wi::STAGE));
    }
  } else {
    // copies NST - 1 = 2 k tiles ahead; g tile kt + 1 routed in LDS during
    // iteration kt, so its pooled row and codes (each thread's first copy of
    // the tile) are waited for one tile ahead and the halo rows (its second,
    // last copy) two tiles ahead.  Loads complete in issue order.
    static_assert(NST == 3 && wi::BK == 2 * wi::IMG, "two halo tiles ahead; a tile is two image rows");
    wi_issue<NST, true>(0, smem, wave, lane, G, X, gc, gbytes, xbytes, p_begin, arow, acol, hrel, hh);
    if (1 < nk) {
      wi_issue<NST, true>(1, smem, wave, lane, G, X, gc, gbytes, xbytes, p_begin, arow, acol, hrel, hh);
      wait_vm<wi::SB>();
    } else {
      wait_vm<0>();
    }
    asm volatile("s_barrier" ::: "memory");
    wi_route(smem, tid, arow, acol);
    for (int kt = 0; kt < nk; ++kt) {
      // tile kt's copies and routed g have landed, and tile kt + 1's pooled
      // row and codes (only its halo copy may still be in flight); every
      // wave is done with tile kt - 1 and with routing tile kt
      if (kt + 1 < nk) wait_vm<1>();
      else wait_vm<0>();
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      asm volatile("s_barrier" ::: "memory");
      // stage (kt + 2) % NST was last read by tile kt - 1 and (its pooled
      // row) by the routing of tile kt - 1
      if (kt + 2 < nk) wi_issue<NST, true>(kt + 2, smem, wave, lane, G, X, gc, gbytes, xbytes, p_begin, arow, acol, hrel, hh);
      // stage (kt + 1) % NST's g tile was last read by tile kt - 2
      if (kt + 1 < nk) wi_route(smem + ((kt + 1) % NST) * wi::STAGE, tid, arow, acol);
      kgroups(lds0 + (uint32_t)((kt % NST) * wi::STAGE));
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  // the second k row's sums to the first's waves through LDS (the stages
  // are free now), one g fragment at a time: 4 waves x 40 floats per lane
  static_assert(4 * 40 * 64 * 4 <= NST * wi::STAGE, "exchange fits the stages");
  float *xch = reinterpret_cast<float *>(smem);
  const int xw = wave & 3;
#pragma unroll
  for (int r2 = 0; r2 < 2; ++r2) {
    __syncthreads();  // (r2 0: every wave is done with the stages; r2 1: with the exchange)
    if (kw == 1) {
#pragma unroll
      for (int i = 0; i < wi::NF; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) xch[((xw * 40 + 4 * i + r) * 64) + lane] = acc[r2][i][r];
#pragma unroll
      for (int r = 0; r < 4; ++r) xch[((xw * 40 + 36 + r) * 64) + lane] = bacc[r2][r];
    }
    __syncthreads();
    if (kw == 0) {
#pragma unroll
      for (int i = 0; i < wi::NF; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[r2][i][r] += xch[((xw * 40 + 4 * i + r) * 64) + lane];
#pragma unroll
      for (int r = 0; r < 4; ++r) bacc[r2][r] += xch[((xw * 40 + 36 + r) * 64) + lane];
    }
  }
  if (kw != 0) return;

  // column of fragment f, lane j: (tap, channel) = (f / 2, 16 (f % 2) + j),
  // i.e. 16 f + j of the 288
  float *dw = a.dw + split * a.dw_ss + rep * a.dw_rs;
#pragma unroll
  for (int r2 = 0; r2 < 2; ++r2) {
    const int wm = 2 * wm2 + r2;
#pragma unroll
    for (int i = 0; i < wi::NF; ++i) {
      const int n = 16 * (9 * wn + i) + j;
#pragma unroll
      for (int r = 0; r < 4; ++r) dw[(int64_t)(wm * 16 + lg * 4 + r) * a.nw + n] = acc[r2][i][r];
    }
    if (do_bias && j == 0) {
#pragma unroll
      for (int r = 0; r < 4; ++r) a.db[split * a.db_ss + rep * a.db_rs + wm * 16 + lg * 4 + r] = bacc[r2][r];
    }
  }
}

// ------------------------------------------------------------ image layer
// dW[co][k] = sum_p g[p][co] A[p][k] and db[co] = sum_p g[p][co] for the image
// layer: 32 output channels, k = (r, s, c) over the 3 x 3 taps of the 3 image
// channels (27 columns, zero-padded to 32; the first 27 are written).  A
// stream: each wave walks groups of 32 pixels of the workgroup's chunk,
// copying the group's g rows (2 KB) into its own double-buffered LDS region
// (no workgroup barrier in the loop), and multiplies transposed fragments
// (four MFMAs per group, two more against ones for the bias).  The group's
// im2col rows (2 KB) are either copied from the gathered rows (IMG3 false),
// or (IMG3: bf16 NHWC images 32 pixels wide, so a group is one image row)
// built in the stage by the wave from the image rows above, at and below
// the group's row (576 bytes, copied with the g rows; zero outside the
// image).  The four waves' sums are added in wave order at the end.
namespace wc {
constexpr int CO = 32, KC = 32, PX = 32;  // output channels, columns, pixels per group
constexpr int ROW = 64;                   // bytes per pixel row of either operand
constexpr int OP = PX * ROW;              // 2 KB per operand and group
constexpr int RAW = 1024;                 // IMG3: three image rows of 192 bytes
template <bool IMG3> constexpr int stage() { return 2 * OP + (IMG3 ? RAW : 0); }  // g rows, im2col rows (, image rows)
template <bool IMG3> constexpr int wave_lds() { return 2 * stage<IMG3>(); }      // two stages per wave
constexpr int BK = 128;                   // chunks are multiples of this
constexpr int IMG_W = 32, IMG_C = 3;      // IMG3: image width and channels
constexpr int VROW = IMG_W * IMG_C * 2 / 16;  // 16-byte pieces per image row (12)
}  // namespace wc

__device__ __forceinline__ void wc_issue(char *dst, const bf16_t *G, const bf16_t *X, uint32_t gbytes,
                                         uint32_t xbytes, int p, int lane) {
  const __amdgpu_buffer_rsrc_t rsg = rsrc(G, gbytes);
  const __amdgpu_buffer_rsrc_t rsx = rsrc(X, xbytes);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint32_t off = (uint32_t)(p * wc::ROW + h * 1024 + lane * 16);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsg, LDS_PTR(dst + h * 1024), 16, off, 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsx, LDS_PTR(dst + wc::OP + h * 1024), 16, off, 0, 0, 0);
  }
}

// IMG3: the group's g rows, and image rows h - 1, h, h + 1 of the group's
// image row (b, h) into the stage's raw region (lane 12 r + v: piece v of row
// h + r - 1; lanes past 36 and rows outside the image read zero)
__device__ __forceinline__ void wc_issue_img3(char *dst, const bf16_t *G, const bf16_t *X, uint32_t gbytes,
                                              uint32_t xbytes, int p, int H, int lane) {
  const __amdgpu_buffer_rsrc_t rsg = rsrc(G, gbytes);
  const __amdgpu_buffer_rsrc_t rsx = rsrc(X, xbytes);
#pragma unroll
  for (int h = 0; h < 2; ++h)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsg, LDS_PTR(dst + h * 1024), 16,
                                             (uint32_t)(p * wc::ROW + h * 1024 + lane * 16), 0, 0, 0);
  const int q = p / wc::IMG_W, b = q / H, h = q - b * H;  // the group's image row
  const int r = lane / wc::VROW, v = lane - r * wc::VROW, hh = h + r - 1;
  const uint32_t off = (lane < 3 * wc::VROW && (unsigned)hh < (unsigned)H)
                           ? (uint32_t)((((int64_t)b * H + hh) * wc::IMG_W * wc::IMG_C + 8 * v) * 2)
                           : kOob;
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsx, LDS_PTR(dst + 2 * wc::OP), 16, off, 0, 0, 0);
}

template <bool IMG3>
__global__ void __launch_bounds__(256)
wgrad_col_kernel(WgradArgs a) {
  constexpr int STAGE = wc::stage<IMG3>();
  __shared__ __attribute__((aligned(1024))) char smem[4 * wc::wave_lds<IMG3>()];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t t = xcd_swizzle(blockIdx.x, (uint32_t)(a.splits * a.C));
  const int split = __builtin_amdgcn_readfirstlane((int)(t % (uint32_t)a.splits));
  const int rep = replica_of(a.rmap, __builtin_amdgcn_readfirstlane((int)(t / (uint32_t)a.splits)));
  const int M = a.Bt * a.H * a.W;
  const int p_begin = split * a.chunk;
  // groups of the chunk; a last partial group reads zeros past the last
  // pixel (the copies' range check), which add nothing
  const int ng = (min(M, p_begin + a.chunk) - p_begin + wc::PX - 1) / wc::PX;
  const bf16_t *G = reinterpret_cast<const bf16_t *>(a.g) + rep * a.g_rs;
  const bf16_t *X = reinterpret_cast<const bf16_t *>(a.x) + rep * a.x_rs;
  const uint32_t gbytes = (uint32_t)((int64_t)M * wc::CO * 2),
                 xbytes = (uint32_t)((int64_t)M * (IMG3 ? wc::IMG_C : wc::KC) * 2);
  char *mine = smem + wave * wc::wave_lds<IMG3>();
  auto issue = [&](char *dst, int p) {
    if constexpr (IMG3)
      wc_issue_img3(dst, G, X, gbytes, xbytes, p, a.H, lane);
    else
      wc_issue(dst, G, X, gbytes, xbytes, p, lane);
  };
  // IMG3: lane (px, kh) builds k = 16 kh .. 16 kh + 15 of pixel px's row;
  // (r, s, c) of k sits at raw row r, pixel px + s - 1, channel c
  const int bpx = lane & 31, bkh = lane >> 5;
  const uint32_t base = (uint32_t)(size_t)LDS_PTR(mine);
  // transposing reads: lane (lg, j) takes pixel rows 8 lg + j / 4 (+4), 16-byte
  // chunk 2 c + half of channel block c, 8-byte half j & 1
  const int j = lane & 15, lg = lane >> 4;
  const int half = (j & 3) >> 1;
  const uint32_t fr = (uint32_t)((8 * lg + (j >> 2)) * wc::ROW + half * 16 + (j & 1) * 8);
  f32x4_t acc[2][2], bacc[2];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    bacc[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int d = 0; d < 2; ++d) acc[c][d] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }
  // this wave's groups: wave, wave + 4, ...
  int i = wave;
  if (i < ng) issue(mine, p_begin + i * wc::PX);
  for (int s = 0; i < ng; i += 4, s ^= 1) {
    const bool next = i + 4 < ng;
    if (next) issue(mine + (s ^ 1) * STAGE, p_begin + (i + 4) * wc::PX);
    // the group's own copies have landed once only the next group's are out
    if (next) {
      if constexpr (IMG3)
        asm volatile("s_waitcnt vmcnt(3)" ::: "memory");
      else
        asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
    } else {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
    if constexpr (IMG3) {
      const uint16_t *raw = reinterpret_cast<const uint16_t *>(mine + s * STAGE + 2 * wc::OP);
      uint32_t h16[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int k = 16 * bkh + e, r = k / 9, sc = (k % 9) / 3, c = k % 3, w = bpx + sc - 1;
        h16[e] = (k < 27 && (unsigned)w < (unsigned)wc::IMG_W) ? (uint32_t)raw[r * wc::IMG_W * wc::IMG_C + w * 3 + c]
                                                                : 0u;
      }
      u32x4 *row = reinterpret_cast<u32x4 *>(mine + s * STAGE + wc::OP + bpx * wc::ROW + bkh * 32);
      row[0] = u32x4{h16[0] | (h16[1] << 16), h16[2] | (h16[3] << 16), h16[4] | (h16[5] << 16),
                     h16[6] | (h16[7] << 16)};
      row[1] = u32x4{h16[8] | (h16[9] << 16), h16[10] | (h16[11] << 16), h16[12] | (h16[13] << 16),
                     h16[14] | (h16[15] << 16)};
    }
    const uint32_t st = base + (uint32_t)(s * STAGE);
    u32x4 ga[2], xb[2];
    read_frag<0, wc::ROW>(ga[0], st + fr);
    read_frag<32, wc::ROW>(ga[1], st + fr);
    read_frag<wc::OP, wc::ROW>(xb[0], st + fr);
    read_frag<wc::OP + 32, wc::ROW>(xb[1], st + fr);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
    for (int c = 0; c < 2; ++c) asm volatile("" : "+v"(ga[c]), "+v"(xb[c]));
    const uint32_t one2 = 0x3F803F80u;  // two bf16 ones
#pragma unroll
    for (int c = 0; c < 2; ++c) {
#pragma unroll
      for (int d = 0; d < 2; ++d) mma(acc[c][d], ga[c], xb[d]);
      mma(bacc[c], ga[c], u32x4{one2, one2, one2, one2});
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  // add the four waves' sums in wave order: each wave stages its 16 + 8
  // values per lane, wave 0 adds and writes the chunk's partial
  __syncthreads();
  float *red = reinterpret_cast<float *>(smem);
#pragma unroll
  for (int c = 0; c < 2; ++c) {
#pragma unroll
    for (int d = 0; d < 2; ++d)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[((wave * 24 + (c * 2 + d) * 4 + r) * 64) + lane] = acc[c][d][r];
#pragma unroll
    for (int r = 0; r < 4; ++r) red[((wave * 24 + 16 + c * 4 + r) * 64) + lane] = bacc[c][r];
  }
  __syncthreads();
  if (wave == 0) {
    float *dw = a.dw + split * a.dw_ss + rep * a.dw_rs;
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int d = 0; d < 2; ++d)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float v = 0.f;
          for (int w = 0; w < 4; ++w) v += red[((w * 24 + (c * 2 + d) * 4 + r) * 64) + lane];
          const int co = c * 16 + lg * 4 + r, k = d * 16 + j;
          if (k < a.nw) dw[(int64_t)co * a.nw + k] = v;
        }
    if (a.db != nullptr && j == 0) {
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float v = 0.f;
          for (int w = 0; w < 4; ++w) v += red[((w * 24 + 16 + c * 4 + r) * 64) + lane];
          a.db[split * a.db_ss + rep * a.db_rs + c * 16 + lg * 4 + r] = v;
        }
    }
  }
}

}  // namespace

bool wgrad_col_ok(int dtype, int Co, int Ci, int taps) {
  return dtype == GCPSL_BF16 && taps == 1 && Co == wc::CO && Ci == wc::KC;
}

hipError_t launch_wgrad_col(const WgradArgs &a, hipStream_t s, std::string *label) {
  const bool img3 = a.taps == 9 && conv_im3_ok(GCPSL_BF16, a.Ci, a.Co, a.H, a.W);
  if (!(img3 || wgrad_col_ok(GCPSL_BF16, a.Co, a.Ci, a.taps)) || a.chunk % wc::BK || a.nw > wc::KC)
    return hipErrorInvalidValue;
  if (label) *label = img3 ? "conv_wgrad<bf16,32x27,w4,img3>" : "conv_wgrad<bf16,32x32,w4,col>";
  if (img3)
    hipLaunchKernelGGL(wgrad_col_kernel<true>, dim3((uint32_t)a.splits * a.C), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(wgrad_col_kernel<false>, dim3((uint32_t)a.splits * a.C), dim3(256), 0, s, a);
  return hipGetLastError();
}

bool wgrad_lds_ok(int dtype, int Co, int Ci) {
  return dtype == GCPSL_BF16 && Co >= 64 && Co % 8 == 0 && Ci % 8 == 0;
}

// Tile configurations: rows (output channels) x columns (im2col columns),
// waves, k tile, stages.  Measured on the 256-channel layers: 32-pixel tiles
// in 4 stages and, separately, reads of the next k group pipelined against
// the MFMAs within a wave were no faster than 64-pixel tiles in 2 stages.
using WgBig = Cfg<256, 256, 2, 4, 64, 2>;
using WgMid = Cfg<128, 256, 2, 4, 64, 2>;
using WgSmall = Cfg<64, 128, 1, 8, 64, 2>;

// Halo mode applies to 16 x 16 images with output channels a multiple of 128
// and input channels a multiple of 64 (taps from the layer input).
constexpr int kHaloStages = 2;
// The image-side client layer: 32 x 32 images, 64 output, 32 input channels.
constexpr int kImgStages = 3;
bool wgrad_img_ok(int Co, int Ci, int H, int W, int taps) {
  return taps == 9 && H == wi::IMG && W == wi::IMG && Co == wi::CO && Ci == wi::CI;
}

bool wgrad_pool_codes(int dtype, int Co, int Ci, int H, int W, int taps) {
  return dtype == GCPSL_BF16 && wgrad_img_ok(Co, Ci, H, W, taps);
}

bool wgrad_halo_ok(int Co, int Ci, int H, int W, int taps) {
  return taps == 9 && H == wh::IMG && W == wh::IMG && Co % wh::BM == 0 && Ci % 64 == 0;
}

// Tile of a layer (rows = output channels, columns of the im2col operand)
// and how many such workgroups one CU holds (LDS-limited; halo mode: one,
// its 8 waves hold 144 accumulator registers per lane).
void wgrad_lds_tile(int Co, int Ci, int H, int W, int taps, int *bm, int *bn, int *bk, int *per_cu) {
  if ((taps == 1 && Co == wc::CO && Ci == wc::KC) || (taps == 9 && conv_im3_ok(GCPSL_BF16, Ci, Co, H, W))) {
    *bm = wc::CO; *bn = wc::KC; *bk = wc::BK; *per_cu = 4;
  } else if (wgrad_halo_ok(Co, Ci, H, W, taps)) {
    *bm = wh::BM; *bn = 9 * 64; *bk = wh::BK; *per_cu = 1;
  } else if (wgrad_img_ok(Co, Ci, H, W, taps)) {
    *bm = wi::CO; *bn = 9 * wi::CI; *bk = wi::BK; *per_cu = 160 * 1024 / (kImgStages * wi::STAGE);
  } else if (Co > 128) {
    *bm = 256; *bn = 256; *bk = WgBig::BK; *per_cu = 160 * 1024 / WgBig::LDS_BYTES;
  } else if (Co > 64) {
    *bm = 128; *bn = 256; *bk = WgMid::BK; *per_cu = 160 * 1024 / WgMid::LDS_BYTES;
  } else {
    *bm = 64; *bn = 128; *bk = WgSmall::BK; *per_cu = 160 * 1024 / WgSmall::LDS_BYTES;
  }
}

// Every instantiation is named in this (non-template) function.
hipError_t launch_wgrad_lds(const WgradArgs &a, hipStream_t s, std::string *label) {
#define WG_K(CF, T) wgrad_lds_kernel<CF::BM_, CF::BN_, CF::WM_, CF::WN_, CF::BK, CF::NST, T>
#define WG_ATTR(CF)                                                                                          \
  for (const void *f : {reinterpret_cast<const void *>(&WG_K(CF, true)),                                    \
                        reinterpret_cast<const void *>(&WG_K(CF, false))}) {                                \
    const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, CF::LDS_BYTES);  \
    if (e != hipSuccess) return e;                                                                           \
  }
  static PerDeviceOnce attr;
  if (attr.needed()) {
    WG_ATTR(WgBig)
    WG_ATTR(WgMid)
    WG_ATTR(WgSmall)
    attr.mark();
  }
  int BM, BN, bk, per_cu;
  wgrad_lds_tile(a.Co, a.Ci, a.H, a.W, a.taps, &BM, &BN, &bk, &per_cu);
  if (a.chunk % bk) return hipErrorInvalidValue;
  if (wgrad_img_ok(a.Co, a.Ci, a.H, a.W, a.taps)) {
    constexpr int lds = kImgStages * wi::STAGE;
    static PerDeviceOnce iattr;
    if (iattr.needed()) {
      for (const void *f : {reinterpret_cast<const void *>(&wgrad_img_kernel<kImgStages, false>),
                            reinterpret_cast<const void *>(&wgrad_img_kernel<kImgStages, true>)}) {
        const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
        if (e != hipSuccess) return e;
      }
      iattr.mark();
    }
    if (label) *label = a.gcode ? "conv_wgrad<bf16,64x288,w8,img,pool>" : "conv_wgrad<bf16,64x288,w8,img>";
    if (a.gcode)
      hipLaunchKernelGGL((wgrad_img_kernel<kImgStages, true>), dim3((uint32_t)a.splits * a.C), dim3(wi::NTHR), lds,
                         s, a);
    else
      hipLaunchKernelGGL((wgrad_img_kernel<kImgStages, false>), dim3((uint32_t)a.splits * a.C), dim3(wi::NTHR), lds,
                         s, a);
    return hipGetLastError();
  }
  if (wgrad_halo_ok(a.Co, a.Ci, a.H, a.W, a.taps)) {
    constexpr int lds = kHaloStages * wh::STAGE;
    static PerDeviceOnce hattr;
    if (hattr.needed()) {
      const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&wgrad_halo_kernel<kHaloStages>),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, lds);
      if (e != hipSuccess) return e;
      hattr.mark();
    }
    const int MT = a.Co / wh::BM, NT = a.Ci / 64;
    if (label) *label = "conv_wgrad<bf16,128x576,w8,halo>";
    hipLaunchKernelGGL((wgrad_halo_kernel<kHaloStages>), dim3((uint32_t)MT * NT * a.splits * a.C), dim3(wh::NTHR),
                       lds, s, a, MT, NT);
    return hipGetLastError();
  }
  const int NW = a.taps == 1 ? a.Ci : 9 * a.Ci;
  const int MT = (a.Co + BM - 1) / BM, NT = (NW + BN - 1) / BN;
  const FastDiv fw = make_fastdiv(a.W), fh = make_fastdiv(a.H), fc = make_fastdiv(a.Ci);
  const dim3 g((uint32_t)MT * NT * a.splits * a.C);
  if (label)
    *label = "conv_wgrad<bf16," + std::to_string(BM) + "x" + std::to_string(BN) + ",w8,lds>";
#define WG_GO(CF, T) hipLaunchKernelGGL((WG_K(CF, T)), g, dim3(CF::NTHR), (CF::LDS_BYTES), s, a, fw, fh, fc, MT, NT)
  const bool t1 = a.taps == 1;
  if (BM == 256) {
    if (t1) WG_GO(WgBig, true); else WG_GO(WgBig, false);
  } else if (BM == 128) {
    if (t1) WG_GO(WgMid, true); else WG_GO(WgMid, false);
  } else {
    if (t1) WG_GO(WgSmall, true); else WG_GO(WgSmall, false);
  }
#undef WG_GO
#undef WG_ATTR
#undef WG_K
  return hipGetLastError();
}
