// Forward and input-gradient (dgrad) 3x3 convolutions, bf16, on gfx950, as
// implicit GEMMs over k = (r, s, c):
//
//   fwd    out[m][n] = ReLU(sum_k x[m + (r-1, s-1)][c] Wf[n][k] + bias[n] (+ res[m][n]))
//   dgrad  dx[m][n]  = (sum_k g[m + (r-1, s-1)][c] Wd[n][k] (+ res[m][n])) * [mask[m][n] > 0]
//
// (dgrad is a forward conv of g with the flipped, transposed weights Wd).
// Both operands are k-contiguous: a k tile (64 values, 128 bytes per row) of
// BM pixel rows (gathered per kernel tap from the NHWC activation) and of BN
// weight rows is copied into LDS by buffer loads that write LDS directly;
// taps outside the image, pixels past the batch and weight rows past N read
// zero through the buffer range check.  Rows are XOR-swizzled in 16-byte
// chunks (chunk ^ ((row >> 1) & 7)) so that the 16 rows of one fragment read
// hit all banks.  The fragment reads are inline asm with explicit lgkmcnt
// waits so the compiler does not wait for every outstanding copy.
//
// The workgroup tile is large (up to 256 pixels x 256 channels) because the
// per-CU vector-memory path, not LDS or the MFMA pipe, bounds a k tile: the
// bytes copied per MFMA fall as the tile grows.  Two LDS stages: the copy of
// tile kt+1 is issued right after the barrier that starts tile kt and has
// all of tile kt's MFMAs to land.
//
// The MFMA takes weight fragments as its A operand and pixel fragments as B,
// so each lane accumulates 4 consecutive output channels of one pixel.  The
// epilogue stages the fp32 tile through LDS, 64 pixel rows per pass, then
// works on 8 consecutive channels per lane: 16-byte loads of the residual and
// mask (all of a pass issued together), 16-byte stores.
//
// Residual layers add the layer input itself (cin == cout).  With 64-channel
// wave tiles and the tap-fastest k order, the centre-tap k tile of channel
// block cb holds exactly input[m][cb*64 .. cb*64+63] for the tile's pixels,
// i.e. the residual of the waves whose channels are block cb: those waves add
// it to their accumulators from LDS, and the epilogue reads no residual from
// HBM (the epilogues of all workgroups run at once and are bandwidth-bound).
#include <utility>

#include "runtime.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define LDS_PTR(p) ((__attribute__((address_space(3))) void *)(p))

constexpr int BK = 64;
constexpr int ROW = BK * 2;  // bytes per LDS row
constexpr uint32_t kOob = 0x80000000u;
constexpr int kBufferFlags = 0x00020000;

template <int BM_, int BN, int WM, int WN, int PFO = 0> struct Cfg {
  static constexpr int BM = BM_, BN_ = BN;
  static constexpr int NW = WM * WN, NTHR = 64 * NW;  // waves, threads
  static constexpr int A_BYTES = BM * ROW, B_BYTES = BN * ROW;
  static constexpr int STAGE = A_BYTES + B_BYTES;
  // copies per thread; a narrow weight tile leaves the last B copy to the
  // first waves only
  static constexpr int SA = A_BYTES / (NTHR * 16), SB = (B_BYTES + NTHR * 16 - 1) / (NTHR * 16);
  static constexpr int TM = BM / WM / 16, TN = BN / WN / 16;  // fragments per wave
  static constexpr int WNW = BN / WN;                          // wave tile width
  // epilogue: PF pixel fragments (16 * PF rows) per pass through LDS
  static constexpr int PF = PFO ? PFO : (NW > 8 ? 2 : 4);
  // floats per staged epilogue row: 64-wide wave tiles use unpadded rows
  // whose 16-byte chunks are XOR-ed with the row's low 3 bits (measured free
  // of LDS bank conflicts for both the fragment writes and the 8-channel
  // reads); narrower tiles pad rows by 4 floats
  static constexpr bool EP_SWZ = WNW == 64;
  static constexpr int EP_LD = EP_SWZ ? WNW : WNW + 4;
  static constexpr int EP_BYTES = NW * 16 * PF * EP_LD * 4;
  static constexpr int LDS_BYTES = 2 * STAGE > EP_BYTES ? 2 * STAGE : EP_BYTES;
  static_assert(NW == 8 || NW == 16, "8 or 16 waves");
  static_assert(SA * NTHR * 16 == A_BYTES && B_BYTES % 1024 == 0, "copies must tile the stage");
  static_assert(TM % PF == 0 && TM % 2 == 0 && TN >= 1, "wave tile: whole epilogue passes, two halves per k group");
  static_assert(LDS_BYTES <= 160 * 1024, "LDS");
};

// Halo mode (16 x 16 images, 256-pixel tiles: one image per tile, 64-channel
// multiples): per 64-channel block the image is staged once with a one-pixel
// zero border, 18 x 18 rows of 128 bytes, and the 9 taps read their pixel
// fragments from it at shifted rows, so a tile's pixels are copied once per
// channel block instead of once per tap.  Row R = 18 h' + w' stores its
// 16-byte chunk c at c ^ hswz(w'), hswz(w') = w' & 7: the 16-row fragment
// reads of all three tap columns (rows R0 .. R0 + 15, R0 = 18 h' + s) are
// then free of LDS bank conflicts (measured with the hardware counter; the
// (w' >> 1) & 7 key cost 4 conflict cycles per read at s = 1, 2), and
// fragments of successive image rows sit a constant 18 rows (2304 bytes)
// apart.  Two halo buffers (by channel block)
// and two weight stages (by k tile).
//
// A 128-wide weight tile (8 waves) keeps one halo buffer: its k loop, two
// weight stages and two-pass epilogue fit in 73 KB, so two workgroups share
// a CU and one's prologue, epilogue and barrier waits overlap the other's
// MFMAs.  With one buffer the next channel block's halo is loaded when the
// last tap of the current block is done (one wait per channel block).
namespace halo {
constexpr int IMG = 16, HP = IMG + 2, ROWS = HP * HP;    // 18 x 18 rows
constexpr int BYTES = ((ROWS * 128 + 1023) / 1024) * 1024;  // padded to whole 1 KB wave copies
constexpr int FSTRIDE = HP * 128;                         // bytes between image-row fragments
// 16-byte copies per thread for a workgroup of NTHR threads
template <int NTHR> constexpr int pieces() { return (ROWS * 128 + NTHR * 16 - 1) / (NTHR * 16); }
// k tiles: TPK kernel taps of one 64-channel block (TPK = 1, or 3 for a whole
// tap row); HB halo buffers and two weight stages of TPK x BN rows
template <int BN, int TPK, int HB = 2> constexpr int lds_bytes() { return HB * BYTES + 2 * TPK * BN * 128; }
static_assert(pieces<1024>() == 3 && pieces<512>() == 6 && lds_bytes<256, 1>() <= 160 * 1024 &&
              lds_bytes<128, 1, 1>() <= 80 * 1024, "halo layout");
}  // namespace halo
__device__ __forceinline__ int hswz(int wp) { return wp & 7; }

__device__ __forceinline__ int swz(int row) { return (row >> 1) & 7; }
__device__ __forceinline__ int wn_of(int wave, int WN) { return wave % WN; }

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

// T fragments 16 rows (2048 bytes) apart; the reads stay in flight.  The
// offsets are template constants (an asm immediate must be one).
template <int OFF>
__device__ __forceinline__ void read_frag(u32x4 &f, uint32_t addr) {
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(f) : "v"(addr), "n"(OFF));
}
template <int T, int START, int STRIDE, int... I>
__device__ __forceinline__ void read_frags_seq(u32x4 (&f)[T], uint32_t addr, std::integer_sequence<int, I...>) {
  (read_frag<(START + I) * STRIDE>(f[I], addr), ...);
}
// fragments START .. START+T-1 of a column of fragments STRIDE bytes apart
// (2048: 16-row blocks)
template <int T, int START = 0, int STRIDE = 2048>
__device__ __forceinline__ void read_frags(u32x4 (&f)[T], uint32_t addr) {
  read_frags_seq<T, START, STRIDE>(f, addr, std::make_integer_sequence<int, T>{});
}

// Wait for every outstanding LDS read, then mark the fragments as produced
// here so that no use of them is scheduled before the wait.
template <int TA, int TB>
__device__ __forceinline__ void wait_frags(u32x4 (&x)[TA], u32x4 (&w)[TB]) {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int t = 0; t < TA; ++t) asm volatile("" : "+v"(x[t]));
#pragma unroll
  for (int t = 0; t < TB; ++t) asm volatile("" : "+v"(w[t]));
}
template <int TA>
__device__ __forceinline__ void wait_frags(u32x4 (&x)[TA]) {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int t = 0; t < TA; ++t) asm volatile("" : "+v"(x[t]));
}

__device__ __forceinline__ float bf2f(uint32_t bits16) { return bf16_to_f32((bf16_t)bits16); }

// Copies of k tile kt into its stage: this thread's SA pixel-row and SB
// weight-row 16-byte pieces.  The buffer resources are built here from plain
// pointers: a buffer-resource value passed into a function or lambda of a
// kernel template makes the host compilation pass drop the kernel's launch
// stub without a diagnostic.
template <typename CF, bool TAPS1>
__device__ __forceinline__ void issue_tile(int kt, char *stage0, int wave, const ConvArgs &a, FastDiv fd_c,
                                           const void *src, const void *wt, const int *achunk, const int *arowoff,
                                           const uint32_t *amask, const uint32_t *boff) {
  const __amdgpu_buffer_rsrc_t rsa = rsrc(src, (uint32_t)(a.src_rs * 2));
  const __amdgpu_buffer_rsrc_t rsb = rsrc(wt, (uint32_t)((int64_t)a.N * a.Kp * 2));
  char *sa = stage0 + (kt & 1) * CF::STAGE;
  int kcol = kt * BK;  // first weight column of the tile
  if (!TAPS1 && a.Csrc % BK == 0) {
    // The whole k tile lies in one kernel tap (tap and offset are
    // workgroup-uniform), and tiles run tap-fastest: k tile kt is channel
    // block kt / 9 of tap kt % 9, so the 9 taps reuse one 64-channel window
    // of pixel rows while it is in L2.
    const int cb = __builtin_amdgcn_readfirstlane(kt / 9);
    const int rs = kt - 9 * cb;
    const int r = (rs * 11) >> 5;  // rs / 3 for rs < 9
    const int tap = __builtin_amdgcn_readfirstlane(((r - 1) * a.W + (rs - 3 * r - 1)) * a.Csrc + cb * BK);
    kcol = rs * a.Csrc + cb * BK;
#pragma unroll
    for (int q = 0; q < CF::SA; ++q) {
      const uint32_t off = ((amask[q] >> rs) & 1u) ? (uint32_t)(arowoff[q] + tap + 8 * achunk[q]) * 2u : kOob;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsa, LDS_PTR(sa + q * CF::NTHR * 16), 16, off, 0, 0, 0);
    }
  } else {
#pragma unroll
    for (int q = 0; q < CF::SA; ++q) {
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
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsa, LDS_PTR(sa + q * CF::NTHR * 16), 16, off, 0, 0, 0);
    }
  }
  const uint32_t kb = (uint32_t)(kcol * 2);
#pragma unroll
  for (int q = 0; q < CF::SB; ++q)
    if (q * CF::NTHR * 16 + wave * 1024 < CF::B_BYTES)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsb, LDS_PTR(sa + CF::A_BYTES + q * CF::NTHR * 16), 16,
                                               boff[q] == kOob ? kOob : boff[q] + kb, 0, 0, 0);
}

// Halo mode: piece q of channel block cb's halo image into buffer cb % HB
// (hoff: this thread's source offset within the image, -1 for the zero
// border); the last piece covers only the first waves.
template <int NTHR, int HB>
__device__ __forceinline__ void issue_halo_piece(int q, int cb, char *smem, int wave, const ConvArgs &a,
                                                 const void *src, int img_off, int hoff) {
  const __amdgpu_buffer_rsrc_t rsa = rsrc(src, (uint32_t)(a.src_rs * 2));
  if (q * NTHR * 16 + wave * 1024 < halo::BYTES) {
    const uint32_t off = hoff >= 0 ? (uint32_t)(img_off + hoff + cb * BK) * 2u : kOob;
    const int buf = HB == 2 ? (cb & 1) : 0;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsa, LDS_PTR(smem + buf * halo::BYTES + q * NTHR * 16 + wave * 1024),
                                             16, off, 0, 0, 0);
  }
}

// Halo mode: the weight rows of k tile kt into weight stage kt % 2: TPK
// taps of channel block kt / (9 / TPK) (one tap kt % 9, or the taps of tap
// row kt % 3), one BN-row sub-stage per tap.
template <typename CF, int TPK, int HB>
__device__ __forceinline__ void issue_weights(int kt, char *smem, int wave, const ConvArgs &a, const void *wt,
                                              const uint32_t *boff) {
  const __amdgpu_buffer_rsrc_t rsb = rsrc(wt, (uint32_t)((int64_t)a.N * a.Kp * 2));
  constexpr int KPB = 9 / TPK;  // k tiles per channel block
  const int cb = kt / KPB, kr = kt - KPB * cb;
  char *sb = smem + HB * halo::BYTES + (kt & 1) * TPK * CF::B_BYTES + wave * 1024;
#pragma unroll
  for (int t = 0; t < TPK; ++t) {
    const int rs = TPK == 1 ? kr : 3 * kr + t;  // kernel tap
    const uint32_t kb = (uint32_t)((rs * a.Csrc + cb * BK) * 2);
#pragma unroll
    for (int q = 0; q < CF::SB; ++q)
      // a narrow stage takes the first waves only
      if (CF::B_BYTES % (CF::NTHR * 16) == 0 || q * CF::NTHR * 16 + wave * 1024 < CF::B_BYTES)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsb, LDS_PTR(sb + t * CF::B_BYTES + q * CF::NTHR * 16), 16,
                                                 boff[q] == kOob ? kOob : boff[q] + kb, 0, 0, 0);
  }
}

// (one halo buffer: at most 128 registers, so that two 8-wave workgroups
// share a CU)
template <int BM, int BN, int WM, int WN, int EPI, bool TAPS1, bool HALO = false, bool AVG = false, int HB = 2>
__global__ void __launch_bounds__(64 * WM * WN, (HALO && HB == 1) ? 4 : 1)
conv_lds_kernel(ConvArgs a, FastDiv fd_w, FastDiv fd_h, FastDiv fd_c, int MT, int NT) {
  // one halo buffer: the two-pass epilogue keeps the staging within the
  // k loop's 73 KB
  using CF = Cfg<BM, BN, WM, WN, (HALO && HB == 1) ? 2 : 0>;
  static_assert(!HALO || (BM == 256 && !TAPS1 &&
                          ((BN == 256 && (WM == 4 || WM == 2) && WN == 4 && HB == 2) ||
                           (BN == 64 && WM == 8 && WN == 2 && HB == 2) ||
                           ((BN == 128 || BN == 64) && WM == 4 && WN == 2 && HB == 1))),
                "halo mode tile");
  static_assert(HB == 2 || (HALO && HB == 1), "halo buffers");
  // AVG: the tile is one whole image (halo mode, forward) and writes the
  // means of its BN channels
  static_assert(!AVG || (HALO && (BN == 256 || BN == 128) && EPI == EPI_FWD), "image mean in the epilogue");
  // halo mode, 64-wide weight tiles with two halo buffers: a k tile is a
  // whole tap row (three taps) so that each barrier covers three times the
  // MFMAs of a one-tap tile
  constexpr int TPK = (HALO && BN == 64 && HB == 2) ? 3 : 1;
  constexpr int SA = CF::SA, SB = CF::SB, TM = CF::TM, TN = CF::TN, NTHR = CF::NTHR, PF = CF::PF;
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t tile = xcd_swizzle(blockIdx.x, (uint32_t)(MT * NT * a.C));
  const int nt = __builtin_amdgcn_readfirstlane((int)(tile % (uint32_t)NT));
  const uint32_t rest = tile / (uint32_t)NT;
  const int mt = __builtin_amdgcn_readfirstlane((int)(rest % (uint32_t)MT));
  const int rep = replica_of(a.rmap, __builtin_amdgcn_readfirstlane((int)(rest / (uint32_t)MT)));
  const int M = a.Bt * a.H * a.W;
  const int m0 = mt * BM, n0 = nt * BN;
  const bf16_t *src = reinterpret_cast<const bf16_t *>(a.src) + rep * a.src_rs;
  const bf16_t *wt = reinterpret_cast<const bf16_t *>(a.wt) + rep * a.wt_rs;

  // This thread's copies: byte q*8192 + wave*1024 + lane*16 of the A (pixel)
  // and B (weight) regions of a stage.  Row and swizzled chunk are fixed;
  // the k tile advances.
  int achunk[SA], arowoff[SA];
  uint32_t amask[SA];  // kernel taps (bit r*3+s) whose source pixel is inside the image
  // halo mode: source offset (pixel of the image x Csrc + chunk column) of
  // this thread's piece q of a halo image, -1 on the zero border
  constexpr int PIECES = halo::pieces<NTHR>();
  int hoff[PIECES];
  if constexpr (HALO) {
#pragma unroll
    for (int q = 0; q < PIECES; ++q) {
      const int g = q * NTHR + tid;  // 16-byte piece: row g / 8, physical chunk g % 8
      const int R = g >> 3, hp = R / halo::HP, wp = R - hp * halo::HP;
      const int c = (g & 7) ^ hswz(wp);
      const bool in = R < halo::ROWS && hp >= 1 && hp <= halo::IMG && wp >= 1 && wp <= halo::IMG;
      hoff[q] = in ? ((hp - 1) * halo::IMG + (wp - 1)) * a.Csrc + 8 * c : -1;
    }
  }
  if constexpr (!HALO) {
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
  }
  uint32_t boff[SB];
#pragma unroll
  for (int q = 0; q < SB; ++q) {
    const int byte = q * NTHR * 16 + wave * 1024 + lane * 16;
    const int row = byte / ROW;
    const int n = n0 + row;
    boff[q] = (n < a.N && byte < CF::B_BYTES) ? ((uint32_t)n * (uint32_t)a.Kp + (uint32_t)(8 * (((byte % ROW) / 16) ^ swz(row)))) * 2u
                      : kOob;
  }

  const int nk = a.Kp / BK / TPK;
  // k tile of the centre tap of this wave's 64-channel block (tap-fastest
  // order: k tile kt is channel block kt / 9, tap kt % 9)
  const int res_kt = ((n0 + wn_of(wave, WN) * CF::WNW) / BK) * 9 + 4;
  char *stage0 = smem + wave * 1024;
  auto issue = [&](int kt) {
    issue_tile<CF, TAPS1>(kt, stage0, wave, a, fd_c, src, wt, achunk, arowoff, amask, boff);
  };

  // fragment read addresses: lane (li, lg) reads row li of a 16-row block,
  // chunk 4*kg + lg; the swizzle depends on li only
  const int li = lane & 15, lg = lane >> 4;
  const int wm = wave / WN, wn = wave % WN;
  const uint32_t lds0 = (uint32_t)(size_t)LDS_PTR(smem);
  uint32_t xa[2], wa[2];
#pragma unroll
  for (int kg = 0; kg < 2; ++kg) {
    const int ph = ((4 * kg + lg) ^ swz(li)) * 16;
    xa[kg] = (uint32_t)((wm * TM * 16 + li) * ROW + ph);
    wa[kg] = (uint32_t)((HALO ? 0 : CF::A_BYTES) + (wn * TN * 16 + li) * ROW + ph);
  }
  // halo mode: the tile is image m0 / 256; its channel block cb sits in halo
  // buffer cb % 2, k tile kt's weights in weight stage kt % 2
  const int img_off = m0 * a.Csrc;
  const int ncb = a.Csrc / BK;
  constexpr int XS = HALO ? halo::FSTRIDE : 2048;  // bytes between pixel fragments

  f32x4_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int k = 0; k < TN; ++k) acc[i][k] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  if constexpr (HALO) {
#pragma unroll
    for (int q = 0; q < PIECES; ++q) issue_halo_piece<NTHR, HB>(q, 0, smem, wave, a, src, img_off, hoff[q]);
    issue_weights<CF, TPK, HB>(0, smem, wave, a, wt, boff);
  } else {
    issue(0);
  }
  for (int kt = 0; kt < nk; ++kt) {
    // own copies of tile kt have landed; after the barrier every wave's
    // have, and every wave is done with tile kt-1, whose stage is refilled
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    asm volatile("s_barrier" ::: "memory");
    uint32_t xb[2], wb;  // pixel fragment bases of the two k groups, weight stage
    uint32_t xst = 0;    // halo mode: the halo buffer of this channel block
    int kr = 0;          // halo mode: k tile within its channel block
    if constexpr (HALO) {
      constexpr int KPB = 9 / TPK;
      const int cb = kt / KPB;
      kr = kt - KPB * cb;
      if constexpr (HB == 1) {
        if (kr == 0 && cb > 0) {
          // every wave is done with channel block cb - 1 (the barrier
          // above): its buffer takes block cb, waited for here
#pragma unroll
          for (int q = 0; q < PIECES; ++q) issue_halo_piece<NTHR, HB>(q, cb, smem, wave, a, src, img_off, hoff[q]);
          asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
          asm volatile("s_barrier" ::: "memory");
        }
      }
      if (kt + 1 < nk) issue_weights<CF, TPK, HB>(kt + 1, smem, wave, a, wt, boff);
      if constexpr (HB == 2) {
        // the next channel block's halo in pieces over the first k tiles (the
        // buffer was last read by channel block cb - 1)
        if (kr < PIECES && cb + 1 < ncb) {
#pragma unroll
          for (int q = 0; q < PIECES; ++q)
            if (q == kr) issue_halo_piece<NTHR, HB>(q, cb + 1, smem, wave, a, src, img_off, hoff[q]);
        }
      }
      xst = lds0 + (uint32_t)((HB == 2 ? (cb & 1) : 0) * halo::BYTES);
      wb = lds0 + (uint32_t)(HB * halo::BYTES + (kt & 1) * TPK * CF::B_BYTES);
      if constexpr (TPK == 1) {
        const int r = (kr * 11) >> 5, sc = kr - 3 * r;  // tap (r, sc)
#pragma unroll
        for (int kg = 0; kg < 2; ++kg)
          xb[kg] = xst + (uint32_t)(((wm * TM + r) * halo::HP + sc + li) * 128 + (((4 * kg + lg) ^ hswz(li + sc)) * 16));
      }
    } else {
      if (kt + 1 < nk) issue(kt + 1);
      wb = lds0 + (uint32_t)((kt & 1) * CF::STAGE);
#pragma unroll
      for (int kg = 0; kg < 2; ++kg) xb[kg] = wb + xa[kg];
    }
    const bool add_res = a.res_lds && kt == res_kt;
#pragma unroll
    for (int t = 0; t < TPK; ++t) {
      uint32_t wbt = wb;  // this tap's weight sub-stage
      if constexpr (HALO && TPK > 1) {
        // tap (kr, t) of the tap row
        wbt = wb + (uint32_t)(t * CF::B_BYTES);
#pragma unroll
        for (int kg = 0; kg < 2; ++kg)
          xb[kg] = xst + (uint32_t)(((wm * TM + kr) * halo::HP + t + li) * 128 + (((4 * kg + lg) ^ hswz(li + t)) * 16));
      }
    // per k group: the second half of the pixel fragments is read while the
    // first half is multiplied
#pragma unroll
    for (int kg = 0; kg < 2; ++kg) {
      constexpr int H = TM / 2;
      u32x4 w[TN], x0[H], x1[H];
      read_frags<TN>(w, wbt + wa[kg]);
      read_frags<H, 0, XS>(x0, xb[kg]);
      wait_frags<H, TN>(x0, w);
      read_frags<H, H, XS>(x1, xb[kg]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int tm = 0; tm < H; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) mma(acc[tm][tn], w[tn], x0[tm]);
      __builtin_amdgcn_sched_barrier(0);
      wait_frags<H>(x1);
#pragma unroll
      for (int tm = 0; tm < H; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) mma(acc[H + tm][tn], w[tn], x1[tm]);
    }
    }  // taps of the k tile
    if (add_res) {
      // residual of fragment (tm, tn): 4 channels tn*16 + lg*4 .. +3 of the
      // block at pixel row wm*TM*16 + tm*16 + li of the centre-tap A tile
      // (halo mode: image row wm*TM + tm, column li, at halo row + 1, + 1)
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
        u32x2 rv[TN];
        const int row = wm * TM * 16 + tm * 16 + li;
        const int hrow = (wm * TM + tm + 1) * halo::HP + li + 1;
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          const int ch = tn * 2 + (lg >> 1);  // 16-byte chunk of the row
          const uint32_t ad = HALO ? xst + (uint32_t)(hrow * 128 + ((ch ^ hswz(li + 1)) * 16) + (lg & 1) * 8)
                                   : wb + (uint32_t)(row * ROW + ((ch ^ swz(row)) * 16) + (lg & 1) * 8);
          asm volatile("ds_read_b64 %0, %1" : "=v"(rv[tn]) : "v"(ad));
        }
        // the values are produced at the wait: keep every use after it
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) asm volatile("" : "+v"(rv[tn]));
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          acc[tm][tn][0] += bf2f(rv[tn][0] & 0xffffu);
          acc[tm][tn][1] += bf2f(rv[tn][0] >> 16);
          acc[tm][tn][2] += bf2f(rv[tn][1] & 0xffffu);
          acc[tm][tn][3] += bf2f(rv[tn][1] >> 16);
        }
      }
    }
  }
  __syncthreads();

  // epilogue: 16 * PF pixel rows of the wave tile per pass, staged as
  // [pixel][channel] fp32, then 8 channels per lane
  constexpr int PR = 16 * PF;        // rows per pass
  constexpr int SEGS = CF::WNW / 8;  // 8-channel segments per row
  constexpr int RSTEP = 64 / SEGS;   // rows per lane step
  constexpr int ITS = PR / RSTEP;    // lane steps per pass
  float *ep = reinterpret_cast<float *>(smem) + wave * PR * CF::EP_LD;
  const int seg = lane % SEGS;
  const int n = n0 + wn * CF::WNW + 8 * seg;
  const bool nok = n < a.N;
  float bias[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) bias[e] = (EPI == EPI_FWD && nok) ? a.bias[rep * a.bias_rs + n + e] : 0.f;
  bf16_t *out = reinterpret_cast<bf16_t *>(a.out) + rep * a.out_rs;
  const bf16_t *res = (a.res && !a.res_lds) ? reinterpret_cast<const bf16_t *>(a.res) + rep * a.out_rs : nullptr;
  const bf16_t *msk = a.mask ? reinterpret_cast<const bf16_t *>(a.mask) + rep * a.out_rs : nullptr;
  const __amdgpu_buffer_rsrc_t rsr = rsrc(res ? res : out, (uint32_t)(a.out_rs * 2));
  const __amdgpu_buffer_rsrc_t rsm = rsrc(msk ? msk : out, (uint32_t)(a.out_rs * 2));
  // dgrad: the mask loads of every pass are issued up front, so their HBM
  // latency is paid once per tile instead of once per pass
  float avs[8];  // AVG: this lane's sums of its 8 channels over its pixel rows (or windows)
#pragma unroll
  for (int e = 0; e < 8; ++e) avs[e] = 0.f;
  float pv[AVG ? ITS : 1][8];  // AVG: the pass's stored values of this lane
  uint4 mvall[TM / PF][ITS];
  if constexpr (EPI == EPI_DGRAD) {
#pragma unroll
    for (int pass = 0; pass < TM / PF; ++pass)
#pragma unroll
      for (int i = 0; i < ITS; ++i) {
        const int m = m0 + wm * TM * 16 + pass * PR + lane / SEGS + RSTEP * i;
        const uint32_t off = (nok && m < M) ? (uint32_t)((int64_t)m * a.N + n) * 2u : kOob;
        mvall[pass][i] = msk ? __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rsm, off, 0, 0))
                             : make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u);
      }
  }
#pragma unroll
  for (int pass = 0; pass < TM / PF; ++pass) {
#pragma unroll
    for (int tm = 0; tm < PF; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
        *reinterpret_cast<f32x4_t *>(ep + (tm * 16 + li) * CF::EP_LD + 4 * ((tn * 4 + lg) ^ (CF::EP_SWZ ? li & 7 : 0))) =
            acc[pass * PF + tm][tn];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // every residual load of the pass is issued before any is used; rows
    // past M (and channels past N) read zero and store nothing
    uint4 rv[ITS];
#pragma unroll
    for (int i = 0; i < ITS; ++i) {
      const int m = m0 + wm * TM * 16 + pass * PR + lane / SEGS + RSTEP * i;
      const uint32_t off = (nok && m < M) ? (uint32_t)((int64_t)m * a.N + n) * 2u : kOob;
      rv[i] = res ? __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rsr, off, 0, 0))
                  : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < ITS; ++i) {
      const int r = lane / SEGS + RSTEP * i;  // pixel row of this pass
      const int m = m0 + wm * TM * 16 + pass * PR + r;
      const int esw = CF::EP_SWZ ? r & 7 : 0;
      const f32x4_t lo = *reinterpret_cast<const f32x4_t *>(ep + r * CF::EP_LD + 4 * ((2 * seg) ^ esw));
      const f32x4_t hi = *reinterpret_cast<const f32x4_t *>(ep + r * CF::EP_LD + 4 * ((2 * seg + 1) ^ esw));
      float v[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      if (res) {
        const uint32_t rw[4] = {rv[i].x, rv[i].y, rv[i].z, rv[i].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[2 * e] += bf2f(rw[e] & 0xffffu);
          v[2 * e + 1] += bf2f(rw[e] >> 16);
        }
      }
      if constexpr (EPI == EPI_FWD) {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = a.no_relu ? v[e] + bias[e] : fmaxf(v[e] + bias[e], 0.f);
      } else {
        // without a mask source every value passes (ones)
        const uint32_t mw[4] = {mvall[pass][i].x, mvall[pass][i].y, mvall[pass][i].z, mvall[pass][i].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (!(bf2f(mw[e] & 0xffffu) > 0.f)) v[2 * e] = 0.f;
          if (!(bf2f(mw[e] >> 16) > 0.f)) v[2 * e + 1] = 0.f;
        }
      }
      uint4 ov;
      ov.x = pack2_bf16(v[0], v[1]);
      ov.y = pack2_bf16(v[2], v[3]);
      ov.z = pack2_bf16(v[4], v[5]);
      ov.w = pack2_bf16(v[6], v[7]);
      // (with the pool's routing codes the output itself is not kept)
      if (nok && m < M && !(AVG && a.pool_code)) *reinterpret_cast<uint4 *>(out + (int64_t)m * a.N + n) = ov;
      if constexpr (AVG) {
        // the stored (bf16-rounded) values, as the pooling reads them back
        const uint32_t ow[4] = {ov.x, ov.y, ov.z, ov.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          pv[i][2 * e] = bf2f(ow[e] & 0xffffu);
          pv[i][2 * e + 1] = bf2f(ow[e] >> 16);
        }
      }
    }
    if constexpr (AVG) {
      // a pass holds two whole image rows (one pooling row); lane step i
      // is row i >> 1, column lane / 8 + 8 (i & 1)
      static_assert(PR == 2 * halo::IMG && RSTEP == 8 && ITS == 4, "pass = one pooling row");
      if (a.pool_max && a.pool_code) {
        // 2 x 2 windows with routing codes: the even-column lane takes its
        // partner's (lane ^ 8) two values and finds the first maximum in
        // row-major window order (strict comparison), adds it and stores its
        // position, 4 where it is not positive.  Window h of the lane: pooled
        // column (lane / 8) / 2 + 4 h of pooled row 2 wm + pass.
        uint32_t cw[2][2] = {{0u, 0u}, {0u, 0u}};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const float t0 = pv[h][e], b0 = pv[2 + h][e];
            const float t1 = __shfl_xor(t0, 8, 64), b1 = __shfl_xor(b0, 8, 64);
            float best = t0;
            uint32_t arg = 0u;
            if (t1 > best) best = t1, arg = 1u;
            if (b0 > best) best = b0, arg = 2u;
            if (b1 > best) best = b1, arg = 3u;
            if (!(best > 0.f)) arg = 4u;
            if ((lane & 8) == 0) avs[e] += best;
            cw[h][e >> 2] |= arg << (8 * (e & 3));
          }
        }
        if ((lane & 8) == 0 && nok) {
          constexpr int PH = halo::IMG / 2;  // pooled side
          const int img = m0 / (halo::IMG * halo::IMG), prow = 2 * wm + pass;
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int pcol = (lane >> 4) + 4 * h;
            *reinterpret_cast<uint2 *>(a.pool_code + rep * a.code_rs +
                                       ((int64_t)(img * PH + prow) * PH + pcol) * a.N + n) =
                make_uint2(cw[h][0], cw[h][1]);
          }
        }
      } else if (a.pool_max) {
        // 2 x 2 windows: the other column of a window is in lane ^ 8; the
        // even-column lane adds the window's maximum
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float c0 = fmaxf(pv[0][e], pv[2][e]), c1 = fmaxf(pv[1][e], pv[3][e]);
          const float w0 = fmaxf(c0, __shfl_xor(c0, 8, 64)), w1 = fmaxf(c1, __shfl_xor(c1, 8, 64));
          if ((lane & 8) == 0) {
            avs[e] += w0;
            avs[e] += w1;
          }
        }
      } else {
#pragma unroll
        for (int i = 0; i < ITS; ++i)
#pragma unroll
          for (int e = 0; e < 8; ++e) avs[e] += pv[i][e];
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  if constexpr (AVG) {
    // mean over the tile's image (or its 2 x 2 windows) per channel: the 8
    // lanes of a channel segment add over lane bits 3..5 (each pair sum is symmetric, so all
    // 8 hold the same total), then the WM waves of a channel range add in
    // wave order through LDS
    static_assert(SEGS == 8, "8 lanes per segment");
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      avs[e] += __shfl_xor(avs[e], 8, 64);
      avs[e] += __shfl_xor(avs[e], 16, 64);
      avs[e] += __shfl_xor(avs[e], 32, 64);
    }
    __syncthreads();  // every wave is done with its staging rows
    float *ps = reinterpret_cast<float *>(smem);  // [WM][BN]
    if (lane < SEGS) {
#pragma unroll
      for (int e = 0; e < 8; ++e) ps[wm * BN + wn * CF::WNW + 8 * lane + e] = avs[e];
    }
    __syncthreads();
    if (tid < BN && n0 + tid < a.N) {
      float sm = 0.f;
#pragma unroll
      for (int w = 0; w < WM; ++w) sm += ps[w * BN + tid];
      const int npos = a.pool_max ? (a.H / 2) * (a.W / 2) : a.H * a.W;
      bf16_t *ho = reinterpret_cast<bf16_t *>(a.pool_out) + rep * a.pool_rs + (int64_t)(m0 / (a.H * a.W)) * a.N;
      ho[n0 + tid] = f32_to_bf16(sm / (float)npos);
    }
  }
}

template <int BM, int BN>
void grid(const ConvArgs &a, int *MT, int *NT) {
  const int M = a.Bt * a.H * a.W;
  *MT = (M + BM - 1) / BM;
  *NT = (a.N + BN - 1) / BN;
}

}  // namespace

bool conv_lds_ok(int dtype, const ConvArgs &a) {
  return dtype == GCPSL_BF16 && a.N % 8 == 0 && a.Csrc % 8 == 0 && a.Kp % BK == 0;
}

// Halo mode wave layout: kHaloWM x 4 waves on the 256 x 256 tile.
constexpr int kHaloWM = 4;
using HaloCfg = Cfg<256, 256, kHaloWM, 4>;
// 64-wide weight tiles: 16 waves of 32 pixels x 32 channels, tap-row k tiles
using Halo64Cfg = Cfg<256, 64, 8, 2>;
// 128-wide weight tiles: 8 waves of 64 x 64, one halo buffer, two-pass
// epilogue; two workgroups per CU
using Halo128Cfg = Cfg<256, 128, 4, 2, 2>;
// the same on 64-wide weight tiles (8 waves of 64 x 32): three LDS reads
// per four MFMAs instead of the 16-wave tile's one per MFMA
using Halo64hCfg = Cfg<256, 64, 4, 2, 2>;
// dynamic LDS of a halo-mode launch: the k loop's buffers or the epilogue's
// staging, whichever is larger
template <typename CF, int TPK, int HB = 2> constexpr int halo_lds_of() {
  return halo::lds_bytes<CF::BN_, TPK, HB>() > CF::EP_BYTES ? halo::lds_bytes<CF::BN_, TPK, HB>() : CF::EP_BYTES;
}
static_assert(halo_lds_of<HaloCfg, 1>() <= 160 * 1024 && halo_lds_of<Halo64Cfg, 3>() <= 160 * 1024 &&
              2 * halo_lds_of<Halo128Cfg, 1, 1>() <= 160 * 1024 && 2 * halo_lds_of<Halo64hCfg, 1, 1>() <= 160 * 1024,
              "halo LDS");

// 16 x 16 images in 64-channel blocks: the halo layouts apply
bool halo_img16(const ConvArgs &a) {
  return a.taps == 9 && a.Csrc % BK == 0 && a.H == halo::IMG && a.W == halo::IMG;
}
// the 128-wide, one-buffer halo tile for N = 128 or 256 (on the 256-channel
// layers of the 16-cluster step: forward 1.38 -> 0.95 + 0.46 ms, input
// gradient 1.40 -> 1.25 ms per step against the 256-wide tile, whose
// workgroup fills a CU)
bool use_halo128(const ConvArgs &a) { return halo_img16(a) && (a.N == 128 || a.N == 256); }

// The halo forward on a 256-wide weight tile writes the per-image channel
// means to pool_out as well when that is set (launch_conv reaches
// launch_conv_lds for these arguments: not an image-side or im2col layer).
bool conv_fuses_avg(int dtype, const ConvArgs &a) {
  return a.epi == EPI_FWD && !conv_img_ok(dtype, a) && conv_lds_ok(dtype, a) && halo_img16(a) && a.N >= 128 &&
         a.N <= 256;
}

// Every instantiation is named in this (non-template) function, which is
// what makes the compiler emit the host-side launch stubs.
hipError_t launch_conv_lds(const ConvArgs &a, hipStream_t s, std::string *label) {
#define CONV_LDS_K(BM, BN, WM, WN, E, T) conv_lds_kernel<BM, BN, WM, WN, E, T>
#define CONV_LDS_ATTR(BM, BN, WM, WN)                                                                   \
  for (const void *f : {reinterpret_cast<const void *>(&CONV_LDS_K(BM, BN, WM, WN, EPI_FWD, false)),       \
                        reinterpret_cast<const void *>(&CONV_LDS_K(BM, BN, WM, WN, EPI_FWD, true)),        \
                        reinterpret_cast<const void *>(&CONV_LDS_K(BM, BN, WM, WN, EPI_DGRAD, false)),     \
                        reinterpret_cast<const void *>(&CONV_LDS_K(BM, BN, WM, WN, EPI_DGRAD, true))}) {   \
    const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize,               \
                                             Cfg<BM, BN, WM, WN>::LDS_BYTES);                             \
    if (e != hipSuccess) return e;                                                                        \
  }
  static PerDeviceOnce attr;
  if (attr.needed()) {
    for (const void *f : {reinterpret_cast<const void *>(&conv_lds_kernel<256, 256, kHaloWM, 4, EPI_FWD, false, true>),
                          reinterpret_cast<const void *>(&conv_lds_kernel<256, 256, kHaloWM, 4, EPI_FWD, false, true, true>),
                          reinterpret_cast<const void *>(&conv_lds_kernel<256, 256, kHaloWM, 4, EPI_DGRAD, false, true>)}) {
      const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, halo_lds_of<HaloCfg, 1>());
      if (e != hipSuccess) return e;
    }
    for (const void *f : {reinterpret_cast<const void *>(&conv_lds_kernel<256, 64, 8, 2, EPI_FWD, false, true>),
                          reinterpret_cast<const void *>(&conv_lds_kernel<256, 64, 8, 2, EPI_DGRAD, false, true>)}) {
      const hipError_t e =
          hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, halo_lds_of<Halo64Cfg, 3>());
      if (e != hipSuccess) return e;
    }
    {
      const hipError_t e =
          hipFuncSetAttribute(reinterpret_cast<const void *>(&conv_lds_kernel<256, 64, 4, 2, EPI_DGRAD, false, true, false, 1>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, halo_lds_of<Halo64hCfg, 1, 1>());
      if (e != hipSuccess) return e;
    }
    for (const void *f :
         {reinterpret_cast<const void *>(&conv_lds_kernel<256, 128, 4, 2, EPI_FWD, false, true, false, 1>),
          reinterpret_cast<const void *>(&conv_lds_kernel<256, 128, 4, 2, EPI_FWD, false, true, true, 1>),
          reinterpret_cast<const void *>(&conv_lds_kernel<256, 128, 4, 2, EPI_DGRAD, false, true, false, 1>)}) {
      const hipError_t e =
          hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, halo_lds_of<Halo128Cfg, 1, 1>());
      if (e != hipSuccess) return e;
    }
    CONV_LDS_ATTR(256, 256, 4, 4)
    CONV_LDS_ATTR(256, 128, 4, 2)
    CONV_LDS_ATTR(128, 64, 2, 4)
    CONV_LDS_ATTR(256, 64, 4, 2)
    CONV_LDS_ATTR(256, 32, 4, 2)
    attr.mark();
  }
  // the narrowest weight tile that covers N (256 beyond 128); a 64-wide
  // tile over a long k loop takes 128 pixels (48 KB of LDS: three
  // workgroups per CU hide more latency), over a short one 256 (less fixed
  // cost per output)
  int bn = a.N > 128 ? 256 : a.N > 64 ? 128 : a.N > 32 ? 64 : 32;
  // halo mode: one 16 x 16 image per 256-pixel tile, 64-channel blocks, with
  // 256-wide weight tiles or (input channels a multiple of 64, no residual)
  // 64-wide ones
  const bool img16 = halo_img16(a);
  const bool use_h128 = use_halo128(a);
  const bool use_halo = img16 && bn == 256 && !use_h128;
  const bool use_halo64 = img16 && bn == 64 && a.res == nullptr;
  int bm = (bn == 64 && a.Kp >= 16 * BK && !use_halo64) ? 128 : 256;
  if (!img16) {
    // a small grid (low-resolution layers of a few replicas: 8 x 8 or 4 x 4
    // maps of 64 examples fill 64 or fewer 256 x 256 tiles) takes narrower
    // tiles, 256 x 128 and then 128 x 64, until about two workgroups per CU
    const int64_t Mr = (int64_t)a.Bt * a.H * a.W;
    auto wgs = [&](int m, int n) { return ((Mr + m - 1) / m) * ((a.N + n - 1) / n) * a.C; };
    if (bn == 256 && wgs(256, 256) < 512) bn = 128;
    if (bn == 128 && wgs(256, 128) < 512) bn = 64, bm = 128;
  }
  int MT, NT;
  if (use_h128) grid<256, 128>(a, &MT, &NT);
  else if (bn == 256) grid<256, 256>(a, &MT, &NT);
  else if (bn == 128) grid<256, 128>(a, &MT, &NT);
  else if (bn == 64 && bm == 128) grid<128, 64>(a, &MT, &NT);
  else if (bn == 64) grid<256, 64>(a, &MT, &NT);
  else grid<256, 32>(a, &MT, &NT);
  const FastDiv fw = make_fastdiv(a.W), fh = make_fastdiv(a.H), fc = make_fastdiv(a.Csrc);
  const dim3 g((uint32_t)MT * NT * a.C);
  // residual from the staged centre tap: residual == input, tap-fastest k
  // order (input channels a multiple of the k tile), 64-channel wave tiles
  ConvArgs b = a;
  b.res_lds = (a.res != nullptr && a.res == a.src && a.taps == 9 && a.Csrc % BK == 0 && a.Csrc == a.N &&
               (bn == 256 || bn == 128)) ? 1 : 0;
  // the input gradient on 64-wide halo tiles: 8 waves, one halo buffer
  const bool use_h64 = use_halo64 && a.epi == EPI_DGRAD;
  if (label) {
    if (use_h128)
      *label = std::string(a.epi == EPI_FWD ? "conv_fwd" : "conv_dgrad") + "<bf16,256x128x64,w8,halo1>";
    else if (use_h64)
      *label = "conv_dgrad<bf16,256x64x64,w8,halo1>";
    else
      *label = std::string(a.epi == EPI_FWD ? "conv_fwd" : "conv_dgrad") + "<bf16," + std::to_string(bm) + "x" +
               std::to_string(bn) + (use_halo64 ? "x192,w16" : "x64,w") +
               (use_halo ? std::to_string(HaloCfg::NW) : use_halo64 ? "" : bn == 256 ? "16" : "8") +
               ((use_halo || use_halo64) ? ",halo>" : ",lds>");
  }
  if (use_h128) {
    // (with the image means: each 128-channel tile writes its own channels')
    const dim3 gh((uint32_t)MT * NT * a.C);
    if (a.epi == EPI_FWD && a.pool_out != nullptr)
      hipLaunchKernelGGL((conv_lds_kernel<256, 128, 4, 2, EPI_FWD, false, true, true, 1>), gh, dim3(Halo128Cfg::NTHR),
                         (halo_lds_of<Halo128Cfg, 1, 1>()), s, b, fw, fh, fc, MT, NT);
    else if (a.epi == EPI_FWD)
      hipLaunchKernelGGL((conv_lds_kernel<256, 128, 4, 2, EPI_FWD, false, true, false, 1>), gh, dim3(Halo128Cfg::NTHR),
                         (halo_lds_of<Halo128Cfg, 1, 1>()), s, b, fw, fh, fc, MT, NT);
    else
      hipLaunchKernelGGL((conv_lds_kernel<256, 128, 4, 2, EPI_DGRAD, false, true, false, 1>), gh,
                         dim3(Halo128Cfg::NTHR), (halo_lds_of<Halo128Cfg, 1, 1>()), s, b, fw, fh, fc, MT, NT);
    return hipGetLastError();
  }
  if (use_halo) {
    if (a.epi == EPI_FWD && a.pool_out != nullptr && NT == 1)
      hipLaunchKernelGGL((conv_lds_kernel<256, 256, kHaloWM, 4, EPI_FWD, false, true, true>), g, dim3(HaloCfg::NTHR),
                         (halo_lds_of<HaloCfg, 1>()), s, b, fw, fh, fc, MT, NT);
    else if (a.epi == EPI_FWD)
      hipLaunchKernelGGL((conv_lds_kernel<256, 256, kHaloWM, 4, EPI_FWD, false, true>), g, dim3(HaloCfg::NTHR),
                         (halo_lds_of<HaloCfg, 1>()), s, b, fw, fh, fc, MT, NT);
    else
      hipLaunchKernelGGL((conv_lds_kernel<256, 256, kHaloWM, 4, EPI_DGRAD, false, true>), g, dim3(HaloCfg::NTHR),
                         (halo_lds_of<HaloCfg, 1>()), s, b, fw, fh, fc, MT, NT);
    return hipGetLastError();
  }
  if (use_h64) {
    hipLaunchKernelGGL((conv_lds_kernel<256, 64, 4, 2, EPI_DGRAD, false, true, false, 1>), g, dim3(Halo64hCfg::NTHR),
                       (halo_lds_of<Halo64hCfg, 1, 1>()), s, b, fw, fh, fc, MT, NT);
    return hipGetLastError();
  }
  if (use_halo64) {
    if (a.epi == EPI_FWD)
      hipLaunchKernelGGL((conv_lds_kernel<256, 64, 8, 2, EPI_FWD, false, true>), g, dim3(Halo64Cfg::NTHR),
                         (halo_lds_of<Halo64Cfg, 3>()), s, b, fw, fh, fc, MT, NT);
    else
      hipLaunchKernelGGL((conv_lds_kernel<256, 64, 8, 2, EPI_DGRAD, false, true>), g, dim3(Halo64Cfg::NTHR),
                         (halo_lds_of<Halo64Cfg, 3>()), s, b, fw, fh, fc, MT, NT);
    return hipGetLastError();
  }
#define CONV_LDS_GO(BM, BN, WM, WN, E, T)                                                                  \
  hipLaunchKernelGGL((CONV_LDS_K(BM, BN, WM, WN, E, T)), g, dim3(Cfg<BM, BN, WM, WN>::NTHR),                 \
                     (Cfg<BM, BN, WM, WN>::LDS_BYTES), s, b, fw, fh, fc, MT, NT)
#define CONV_LDS_SEL(BM, BN, WM, WN)                                                                        \
  if (fwd) { if (t1) CONV_LDS_GO(BM, BN, WM, WN, EPI_FWD, true); else CONV_LDS_GO(BM, BN, WM, WN, EPI_FWD, false); } \
  else { if (t1) CONV_LDS_GO(BM, BN, WM, WN, EPI_DGRAD, true); else CONV_LDS_GO(BM, BN, WM, WN, EPI_DGRAD, false); }
  const bool fwd = a.epi == EPI_FWD, t1 = a.taps == 1;
  if (bn == 256) { CONV_LDS_SEL(256, 256, 4, 4) }
  else if (bn == 128) { CONV_LDS_SEL(256, 128, 4, 2) }
  else if (bn == 64 && bm == 128) { CONV_LDS_SEL(128, 64, 2, 4) }
  else if (bn == 64) { CONV_LDS_SEL(256, 64, 4, 2) }
  else { CONV_LDS_SEL(256, 32, 4, 2) }
#undef CONV_LDS_SEL
#undef CONV_LDS_GO
#undef CONV_LDS_ATTR
#undef CONV_LDS_K
  return hipGetLastError();
}
