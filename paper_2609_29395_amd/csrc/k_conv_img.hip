// Forward and input-gradient 3x3 convolution of the 32 x 32 image layers with
// 32 or 64 input and output channels, bf16, on gfx950 (the layers between the
// image layer and the cut in the workloads' client segment).
//
//   out[p][n] = epi( sum_{tap, c} src[p + tap][c] * wt[n][tap * Cs + c] )
//
// These layers are bound by HBM, not by the matrix cores: per pixel they read
// Cs and write N channels for 2 * 9 * Cs * N FLOP.  A workgroup takes eight
// full image rows (256 pixels) and every output channel; it copies the ten
// image rows around them with a one-pixel zero border (10 x 34 pixel rows of
// Cs channels) and the layer's whole weight matrix into LDS once, so every
// input pixel crosses the copy path once per workgroup instead of once per
// tap, and computes all nine taps from LDS.  LDS holds two such workgroups
// per CU (42, 62 or 79 KB for 32/32, 32/64 and 64/32 channels), so one
// workgroup's copies overlap the other's MFMAs and stores.
//
// The MFMA takes the weights as A (16 output channels x 32 k) and the pixels
// as B (32 k x 16 pixels), so each lane ends with 4 consecutive channels of
// one pixel; the epilogue regroups them through LDS into whole pixel rows
// and, when the layer is followed by a 2 x 2 max pool, also writes the
// pooled rows (a tile's eight image rows hold four whole pooling rows), and
// then, given a code buffer, the pool's routing codes in place of the
// unpooled rows.  The input gradient of such a layer starts from the pooled
// gradient: its halo pieces are loaded with their codes into registers and
// written to LDS routed (the gradient where the code names the pixel's
// window position, zero elsewhere).  Halo row R (pixel column w'
// of its image row) keeps its 16-byte chunk c at c ^ (w' mod chunks per
// row); weight row n keeps chunk kc at kc ^ (n & 7) (eight-chunk groups).
#include "runtime.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define LDS_PTR(p) ((__attribute__((address_space(3))) void *)(p))

constexpr uint32_t kOob = 0x80000000u;
constexpr int kBufferFlags = 0x00020000;

constexpr int IMG = 32;                    // image side
constexpr int HP = IMG + 2;                // halo row width
constexpr int NTHR = 512;                  // 8 waves: wave w computes image rows RPW w .. RPW w + RPW - 1

// RPW image rows per wave: a tile of 8 RPW image rows (256 RPW pixels)
template <int CS, int NO, int RPW = 1> struct ImgCfg {
  static constexpr int TROWS = 8 * RPW;                          // image rows per workgroup tile
  static constexpr int HR = TROWS + 2, HPIX = HR * HP;           // halo image rows, halo pixels
  static constexpr int RB = CS * 2;                              // bytes per halo pixel row
  static constexpr int CPR = RB / 16;                            // 16-byte chunks per halo row
  static constexpr int H_BYTES = ((HPIX * RB + 1023) / 1024) * 1024;
  static constexpr int KP = ((9 * CS + 63) / 64) * 64;           // weight row length (elements)
  static constexpr int WCH = KP / 8;                             // 16-byte chunks per weight row
  static constexpr int W_BYTES = NO * KP * 2;
  static constexpr int LDS = H_BYTES + W_BYTES;
  static constexpr int HQ = (H_BYTES + NTHR * 16 - 1) / (NTHR * 16);  // halo copies per thread
  static constexpr int WQ = (W_BYTES + NTHR * 16 - 1) / (NTHR * 16);  // weight copies per thread
  static constexpr int TN = NO / 16;                             // output-channel fragments
  static constexpr int KG = CS / 32;                             // 32-channel k groups per tap
  static_assert(CS == 32 || CS == 64, "input channels");
  static_assert(NO == 32 || NO == 64, "output channels");
  static_assert(W_BYTES % 1024 == 0 && WCH % 8 == 0, "weight rows in whole 1 KB copies, 8-chunk groups");
  static constexpr bool FITS2 = 2 * LDS <= 160 * 1024;  // two workgroups per CU
};

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

__device__ __forceinline__ float bf2f(uint32_t bits16) { return bf16_to_f32((bf16_t)bits16); }

// (two rows per wave: at least four waves per SIMD, i.e. at most 128
// registers, so that two workgroups share a CU)
template <int CS, int NO, int EPI, int RPW = 1>
__global__ void __launch_bounds__(NTHR, RPW == 2 ? 4 : 1)
conv_img_kernel(ConvArgs a, int MT) {
  using CF = ImgCfg<CS, NO, RPW>;
  constexpr int TROWS = CF::TROWS, HPIX = CF::HPIX;
  constexpr int TN = CF::TN, KG = CF::KG;
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t t = xcd_swizzle(blockIdx.x, (uint32_t)(MT * a.C));
  const int mt = __builtin_amdgcn_readfirstlane((int)(t % (uint32_t)MT));
  const int rep = replica_of(a.rmap, __builtin_amdgcn_readfirstlane((int)(t / (uint32_t)MT)));
  const int M = a.Bt * IMG * IMG;
  const int m0 = mt * (TROWS * IMG);         // first pixel of the tile
  const int h0 = (m0 / IMG) % IMG;           // its image row (a multiple of 8)
  const bf16_t *src = reinterpret_cast<const bf16_t *>(a.src) + rep * a.src_rs;
  const bf16_t *wt = reinterpret_cast<const bf16_t *>(a.wt) + rep * a.wt_rs;

  // ---- copies: halo image and weight matrix, 16 bytes per lane, LDS-direct;
  // dgrad from a pooled gradient: the halo pieces are routed through the
  // pool's codes in registers and written to the same LDS slots
  const bool pooled = EPI == EPI_DGRAD && a.pool_code != nullptr;
  u32x4 gv[CF::HQ];  // pooled: gradient piece, its 8 codes, window position
  u32x2 cv[CF::HQ];
  int kw[CF::HQ];
  {
    const __amdgpu_buffer_rsrc_t rss = rsrc(src, (uint32_t)((int64_t)M * CS * 2));
    const __amdgpu_buffer_rsrc_t rsw = rsrc(wt, (uint32_t)CF::W_BYTES);
    const uint8_t *cd = pooled ? a.pool_code + rep * a.src_rs : nullptr;
    const int img0 = m0 / (IMG * IMG) * (IMG / 2) * (IMG / 2);  // first pooled pixel of the tile's image
#pragma unroll
    for (int q = 0; q < CF::HQ; ++q) {
      const int byte = q * NTHR * 16 + wave * 1024;  // this wave's 1 KB of the halo region
      kw[q] = -1;
      if (byte < CF::H_BYTES) {
        const int j = byte / 16 + lane;  // 16-byte slot
        const int R = j / CF::CPR, cs = j % CF::CPR;
        const int hp = R / HP, wp = R - hp * HP;
        const int c = cs ^ (wp & (CF::CPR - 1));
        const int h = h0 - 1 + hp, w = wp - 1;
        const bool ok = R < HPIX && (unsigned)h < (unsigned)IMG && (unsigned)w < (unsigned)IMG;
        if (pooled) {
          gv[q] = u32x4{0u, 0u, 0u, 0u};
          cv[q] = u32x2{0u, 0u};
          if (ok) {
            const int pp = (img0 + (h >> 1) * (IMG / 2) + (w >> 1)) * CS + 8 * c;
            gv[q] = *reinterpret_cast<const u32x4 *>(src + pp);
            cv[q] = *reinterpret_cast<const u32x2 *>(cd + pp);
            kw[q] = ((h & 1) << 1) | (w & 1);
          }
        } else {
          const uint32_t off = ok ? (uint32_t)((m0 + (hp - 1) * IMG + w) * CS + 8 * c) * 2u : kOob;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rss, LDS_PTR(smem + byte), 16, off, 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int q = 0; q < CF::WQ; ++q) {
      const int byte = q * NTHR * 16 + wave * 1024;
      if (byte < CF::W_BYTES) {
        const int j = byte / 16 + lane;
        const int row = j / CF::WCH, cs = j % CF::WCH;
        const int kc = cs ^ (row & 7);
        const uint32_t off = (uint32_t)(row * CF::KP + 8 * kc) * 2u;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsw, LDS_PTR(smem + CF::H_BYTES + byte), 16, off, 0, 0, 0);
      }
    }
  }
  if (pooled) {
    // value e of a piece passes where its code names this pixel's window
    // position (a zero-border or out-of-image slot keeps kw = -1: zeros)
#pragma unroll
    for (int q = 0; q < CF::HQ; ++q) {
      const int byte = q * NTHR * 16 + wave * 1024;
      if (byte < CF::H_BYTES) {
        const uint32_t k = (uint32_t)kw[q];
        u32x4 v;
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          const uint32_t cb = cv[q][d >> 1] >> (16 * (d & 1));  // codes of channels 2d, 2d + 1
          const uint32_t keep = ((cb & 0xffu) == k ? 0x0000ffffu : 0u) | (((cb >> 8) & 0xffu) == k ? 0xffff0000u : 0u);
          v[d] = gv[q][d] & keep;
        }
        *reinterpret_cast<u32x4 *>(smem + byte + lane * 16) = v;
      }
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  // ---- nine taps x KG k groups from LDS: wave = image rows RPW wave ..
  // RPW wave + RPW - 1 of the tile; pixel fragment tm = 2 rr + half is
  // pixels 16 half .. 16 half + 15 of row rr
  constexpr int TMW = 2 * RPW;  // pixel fragments per wave
  const int li = lane & 15, lg = lane >> 4;
  const uint32_t lds0 = (uint32_t)(size_t)LDS_PTR(smem);
  f32x4_t acc[TMW][TN];
#pragma unroll
  for (int i = 0; i < TMW; ++i)
#pragma unroll
    for (int k = 0; k < TN; ++k) acc[i][k] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int tap = 0; tap < 9; ++tap) {
    const int r = tap / 3, s = tap % 3;
#pragma unroll
    for (int g = 0; g < KG; ++g) {
      u32x4 w[TN], x[TMW];
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int row = tn * 16 + li;
        const int kc = (tap * CS + g * 32) / 8 + lg;
        const uint32_t ad = lds0 + (uint32_t)(CF::H_BYTES + row * CF::KP * 2 + ((kc ^ (row & 7)) * 16));
        asm volatile("ds_read_b128 %0, %1" : "=v"(w[tn]) : "v"(ad));
      }
#pragma unroll
      for (int tm = 0; tm < TMW; ++tm) {
        const int wp = (tm & 1) * 16 + li + s;
        const int R = (RPW * wave + (tm >> 1) + r) * HP + wp;
        const uint32_t ad = lds0 + (uint32_t)(R * CF::RB + (((4 * g + lg) ^ (wp & (CF::CPR - 1))) * 16));
        asm volatile("ds_read_b128 %0, %1" : "=v"(x[tm]) : "v"(ad));
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
      for (int i = 0; i < TN; ++i) asm volatile("" : "+v"(w[i]));
#pragma unroll
      for (int i = 0; i < TMW; ++i) asm volatile("" : "+v"(x[i]));
#pragma unroll
      for (int tm = 0; tm < TMW; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) mma(acc[tm][tn], w[tn], x[tm]);
    }
  }

  // ---- epilogue: lane holds channels tn*16 + 4*lg .. +3 of pixel tm*16 + li
  // of the wave's rows.  The wave's 32 RPW x NO bf16 results are staged in LDS
  // (its own 32 RPW-row region, 16-byte chunk c of pixel row p at c ^ (p mod
  // chunks per row)) and read back as 16-byte pieces, so every store
  // instruction writes 8 (NO=64) or 16 (NO=32) whole pixel rows, 1 KB
  // contiguous.
  constexpr int OCH = NO / 8;             // 16-byte chunks per output pixel row
  constexpr int OROW = NO * 2;            // bytes per output pixel row
  bf16_t *out = reinterpret_cast<bf16_t *>(a.out) + rep * a.out_rs;
  const int pbase = m0 + wave * RPW * IMG;  // first pixel of this wave's image rows
  const uint32_t stg = lds0 + (uint32_t)(wave * RPW * IMG * OROW);
  float bias[TN][4];
#pragma unroll
  for (int tn = 0; tn < TN; ++tn)
#pragma unroll
    for (int e = 0; e < 4; ++e)
      bias[tn][e] = EPI == EPI_FWD ? a.bias[rep * a.bias_rs + tn * 16 + 4 * lg + e] : 0.f;
  __syncthreads();  // every wave is done with the halo and weight tiles
#pragma unroll
  for (int tm = 0; tm < TMW; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float y = acc[tm][tn][e] + bias[tn][e];
        v[e] = (EPI == EPI_FWD && !a.no_relu) ? fmaxf(y, 0.f) : y;
      }
      u32x2 o;
      o[0] = pack2_bf16(v[0], v[1]);
      o[1] = pack2_bf16(v[2], v[3]);
      const int px = tm * 16 + li, c = 2 * tn + (lg >> 1);
      const uint32_t ad = stg + (uint32_t)(px * OROW + ((c ^ (px & (OCH - 1))) * 16) + (lg & 1) * 8);
      asm volatile("ds_write_b64 %0, %1" ::"v"(ad), "v"(o) : "memory");
    }
  // With one row per wave the max pool reads the neighbouring wave's row
  // too: every wave's staged rows must have landed before the barrier (the
  // compiler does not count the asm writes, so the barrier alone does not
  // wait for them).
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __syncthreads();
  // dgrad: ReLU mask of the layer below (value > 0), read in the same
  // 16-byte pieces; without a mask source every value passes
  const bf16_t *msk = (EPI == EPI_DGRAD && a.mask) ? reinterpret_cast<const bf16_t *>(a.mask) + rep * a.out_rs
                                                   : nullptr;
  constexpr int QN = RPW * IMG * OCH / 64;  // pieces per lane
  u32x4 mv[QN];
#pragma unroll
  for (int q = 0; q < QN; ++q) {
    const int i2 = q * 64 + lane, px = i2 / OCH, c = i2 % OCH;
    mv[q] = msk ? *reinterpret_cast<const u32x4 *>(msk + (int64_t)(pbase + px) * NO + 8 * c)
                : u32x4{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u};
  }
  // forward with pool codes: only the pool and its codes are written
  const bool unpooled = !(EPI == EPI_FWD && a.pool_out && a.pool_code);
#pragma unroll
  for (int q = 0; q < QN; ++q) {
    if (!unpooled) break;
    const int i2 = q * 64 + lane, px = i2 / OCH, c = i2 % OCH;
    u32x4 v;
    const uint32_t ad = stg + (uint32_t)(px * OROW + ((c ^ (px & (OCH - 1))) * 16));
    asm volatile("ds_read_b128 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(ad) : "memory");
    if constexpr (EPI == EPI_DGRAD) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t mlo = mv[q][e] & 0xffffu, mhi = mv[q][e] >> 16;
        const uint32_t keep = (bf2f(mlo) > 0.f ? 0x0000ffffu : 0u) | (bf2f(mhi) > 0.f ? 0xffff0000u : 0u);
        v[e] &= keep;
      }
    }
    *reinterpret_cast<u32x4 *>(out + (int64_t)(pbase + px) * NO + 8 * c) = v;
  }
  if (EPI == EPI_FWD && a.pool_out) {
   // 2 x 2 max pool, one 16-byte channel chunk per lane (the maximum of bf16
   // values is exact).  One row per wave: waves 2k and 2k+1 hold image rows
   // h0+2k, h0+2k+1 and each takes 8 of the 16 pooled pixels of pooled row
   // h0/2 + k.  Two rows per wave: wave k holds both rows of pooled row
   // h0/2 + k and takes its 16 pooled pixels, 8 per pass.
#pragma unroll
   for (int ps = 0; ps < RPW; ++ps) {
    const int pw = (RPW == 1 ? (wave & 1) * 8 : ps * 8) + lane / OCH, c = lane % OCH;
    if (lane < 8 * OCH) {
      const uint32_t r0 = RPW == 1 ? lds0 + (uint32_t)((wave & ~1) * IMG * OROW) : stg;
      const uint32_t r1 = r0 + (uint32_t)(IMG * OROW);
      u32x4 q4[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int px = 2 * pw + (e & 1);
        const uint32_t ad = ((e >> 1) ? r1 : r0) + (uint32_t)(px * OROW + ((c ^ (px & (OCH - 1))) * 16));
        asm volatile("ds_read_b128 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(q4[e]) : "v"(ad) : "memory");
      }
      // window position e = 2 dh + dw (row-major); the first maximum under
      // strict comparison, code 4 where it is not positive
      u32x4 z;
      u32x2 code = u32x2{0u, 0u};
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        uint32_t lo = q4[0][d] & 0xffffu, hi = q4[0][d] >> 16, alo = 0u, ahi = 0u;
#pragma unroll
        for (int e = 1; e < 4; ++e) {
          const uint32_t l2 = q4[e][d] & 0xffffu, h2 = q4[e][d] >> 16;
          if (bf2f(l2) > bf2f(lo)) lo = l2, alo = (uint32_t)e;
          if (bf2f(h2) > bf2f(hi)) hi = h2, ahi = (uint32_t)e;
        }
        z[d] = lo | (hi << 16);
        if (!(bf2f(lo) > 0.f)) alo = 4u;
        if (!(bf2f(hi) > 0.f)) ahi = 4u;
        code[d >> 1] |= (alo | (ahi << 8)) << (16 * (d & 1));
      }
      bf16_t *zo = reinterpret_cast<bf16_t *>(a.pool_out) + rep * a.pool_rs;
      const int b = m0 / (IMG * IMG), hz = h0 / 2 + (RPW == 1 ? (wave >> 1) : wave);
      const int64_t zi = ((int64_t)(b * (IMG / 2) + hz) * (IMG / 2) + pw) * NO + 8 * c;
      *reinterpret_cast<u32x4 *>(zo + zi) = z;
      if (a.pool_code) *reinterpret_cast<u32x2 *>(a.pool_code + rep * a.pool_rs + zi) = code;
    }
   }
  }
}

// The image layer: out[p][n] = act(bias[n] + sum_k A[p][k] W[n][k]) with k =
// (r, s, c) over the 3 x 3 taps of the 3 image channels (27 columns,
// zero-padded to 32) and 32 output channels.  A plain stream: each wave takes
// four groups of 16 pixels, multiplies their rows by the weight fragments it
// keeps in registers (two MFMAs per group) and regroups the results through
// LDS into whole 64-byte output rows.  The rows come either from the
// gathered im2col rows (IMG3 false: one 16-byte piece per lane), or (IMG3)
// from the bf16 NHWC images themselves: a workgroup's 256 pixels are 8 rows
// of one 32-pixel-wide image, whose 10 input rows (one above, one below)
// are staged once in LDS with a zero border, and lane (li, lg) collects its
// 8 values k = 8 lg .. 8 lg + 7 of pixel li from there.
constexpr int COL_K = 32, COL_N = 32, COL_PX = 256;  // k, n, pixels per workgroup
namespace im3 {
constexpr int CIN = 3, W = 32, ROWS = COL_PX / W;   // image channels, width, output rows per workgroup
constexpr int RS = (W + 2) * CIN;                   // bf16 values per staged row (zero pixel either side)
constexpr int LROWS = ROWS + 2;                     // staged rows: one above and one below
constexpr int VROW = W * CIN * 2 / 16;              // 16-byte vectors per image row (12)
}  // namespace im3

template <bool IMG3>
__global__ void __launch_bounds__(256)
conv_col_kernel(ConvArgs a, int MT) {
  __shared__ __attribute__((aligned(16))) char stg_all[4 * 64 * COL_N * 2];
  __shared__ __attribute__((aligned(16))) uint16_t img[IMG3 ? im3::LROWS * im3::RS : 2];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t t = xcd_swizzle(blockIdx.x, (uint32_t)(MT * a.C));
  const int mt = __builtin_amdgcn_readfirstlane((int)(t % (uint32_t)MT));
  const int rep = replica_of(a.rmap, __builtin_amdgcn_readfirstlane((int)(t / (uint32_t)MT)));
  const int M = a.Bt * a.H * a.W;
  const int p0 = mt * COL_PX + wave * 64;  // this wave's 64 pixels
  const int li = lane & 15, lg = lane >> 4;
  const bf16_t *src = reinterpret_cast<const bf16_t *>(a.src) + rep * a.src_rs;
  const bf16_t *wt = reinterpret_cast<const bf16_t *>(a.wt) + rep * a.wt_rs;
  // pixel rows (B operand: lane (li, lg) = pixel li, k 8 lg .. 8 lg + 7)
  u32x4 x[4];
  if constexpr (IMG3) {
    // staged rows h0 - 1 .. h0 + 8 of the tile's image, pixels -1 .. 32
    const int tpi = a.H / im3::ROWS;  // tiles per image
    const int b = mt / tpi, h0 = (mt - b * tpi) * im3::ROWS;
    for (int e = threadIdx.x; e < im3::LROWS * im3::RS / 2; e += 256) reinterpret_cast<uint32_t *>(img)[e] = 0u;
    __syncthreads();
    if (threadIdx.x < im3::LROWS * im3::VROW) {
      const int lr = threadIdx.x / im3::VROW, v = threadIdx.x - lr * im3::VROW, h = h0 - 1 + lr;
      if ((unsigned)h < (unsigned)a.H) {
        const u32x4 q = *reinterpret_cast<const u32x4 *>(src + ((int64_t)b * a.H + h) * im3::W * im3::CIN + 8 * v);
        uint16_t *d = img + lr * im3::RS + im3::CIN + 8 * v;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          d[2 * e] = (uint16_t)(q[e] & 0xffffu);
          d[2 * e + 1] = (uint16_t)(q[e] >> 16);
        }
      }
    }
    __syncthreads();
    // k = 9 r + 3 s + c sits at (row + r) * RS + (pixel + s) * 3 + c =
    // base + k + (RS - 9) r; k >= 27 is padding
    int off[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int k = 8 * lg + e;
      off[e] = k < 27 ? k + (im3::RS - 9) * (k / 9) : -1;
    }
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int pl = wave * 64 + g * 16 + li;  // pixel of the tile: row pl / 32, column pl % 32
      const int base = (pl / im3::W) * im3::RS + (pl % im3::W) * im3::CIN;
      uint32_t h16[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) h16[e] = off[e] >= 0 ? (uint32_t)img[base + off[e]] : 0u;
      x[g] = u32x4{h16[0] | (h16[1] << 16), h16[2] | (h16[3] << 16), h16[4] | (h16[5] << 16),
                   h16[6] | (h16[7] << 16)};
    }
  } else {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int p = p0 + g * 16 + li;
      x[g] = p < M ? *reinterpret_cast<const u32x4 *>(src + (int64_t)p * COL_K + 8 * lg) : u32x4{0u, 0u, 0u, 0u};
    }
  }
  // weights (A operand: lane (li, lg) = output channel tn*16 + li, k 8 lg ..)
  u32x4 w[2];
  float bias[2][4];
#pragma unroll
  for (int tn = 0; tn < 2; ++tn) {
    w[tn] = *reinterpret_cast<const u32x4 *>(wt + (int64_t)(tn * 16 + li) * a.Kp + 8 * lg);
#pragma unroll
    for (int e = 0; e < 4; ++e) bias[tn][e] = a.bias[rep * a.bias_rs + tn * 16 + 4 * lg + e];
  }
  f32x4_t acc[4][2];
#pragma unroll
  for (int g = 0; g < 4; ++g)
#pragma unroll
    for (int tn = 0; tn < 2; ++tn) {
      acc[g][tn] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      mma(acc[g][tn], w[tn], x[g]);
    }
  // lane holds channels tn*16 + 4 lg .. +3 of pixel g*16 + li; stage the
  // wave's 64 x 32 bf16 block (row p, 16-byte chunk c at c ^ (p & 3))
  char *stg = stg_all + wave * 64 * COL_N * 2;
#pragma unroll
  for (int g = 0; g < 4; ++g)
#pragma unroll
    for (int tn = 0; tn < 2; ++tn) {
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float y = acc[g][tn][e] + bias[tn][e];
        v[e] = a.no_relu ? y : fmaxf(y, 0.f);
      }
      u32x2 o;
      o[0] = pack2_bf16(v[0], v[1]);
      o[1] = pack2_bf16(v[2], v[3]);
      const int px = g * 16 + li, c = 2 * tn + (lg >> 1);
      *reinterpret_cast<u32x2 *>(stg + px * 64 + ((c ^ (px & 3)) * 16) + (lg & 1) * 8) = o;
    }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  bf16_t *out = reinterpret_cast<bf16_t *>(a.out) + rep * a.out_rs;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int i2 = q * 64 + lane, px = i2 >> 2, c = i2 & 3;
    const u32x4 v = *reinterpret_cast<const u32x4 *>(stg + px * 64 + ((c ^ (px & 3)) * 16));
    if (p0 + px < M) *reinterpret_cast<u32x4 *>(out + (int64_t)(p0 + px) * COL_N + 8 * c) = v;
  }
}

}  // namespace

bool conv_col_ok(int dtype, const ConvArgs &a) {
  return dtype == GCPSL_BF16 && a.taps == 1 && a.Csrc == COL_K && a.N == COL_N && a.res == nullptr &&
         !a.no_relu && a.Kp >= COL_K && a.Kp % 8 == 0 && ((int64_t)a.Bt * a.H * a.W) % COL_PX == 0;
}

bool conv_im3_ok(int dtype, int Ci, int Co, int H, int W) {
  return dtype == GCPSL_BF16 && Ci == im3::CIN && Co == COL_N && W == im3::W && H % im3::ROWS == 0;
}

hipError_t launch_conv_col(const ConvArgs &a, hipStream_t s, std::string *label) {
  const bool img3 = a.taps == 9 && conv_im3_ok(GCPSL_BF16, a.Csrc, a.N, a.H, a.W);
  if (a.epi != EPI_FWD || a.res != nullptr || a.Kp < COL_K || a.Kp % 8 != 0 ||
      !(img3 || conv_col_ok(GCPSL_BF16, a)))
    return hipErrorInvalidValue;
  const int MT = a.Bt * a.H * a.W / COL_PX;
  if (label) *label = img3 ? "conv_fwd<bf16,256x32x27,w4,img3>" : "conv_fwd<bf16,256x32x32,w4,col>";
  if (img3)
    hipLaunchKernelGGL(conv_col_kernel<true>, dim3((uint32_t)MT * a.C), dim3(256), 0, s, a, MT);
  else
    hipLaunchKernelGGL(conv_col_kernel<false>, dim3((uint32_t)MT * a.C), dim3(256), 0, s, a, MT);
  return hipGetLastError();
}

bool conv_fuses_pool(int dtype, const ConvArgs &a) { return a.epi == EPI_FWD && conv_img_ok(dtype, a); }

bool conv_pool_codes(int dtype, const ConvArgs &a) { return conv_img_ok(dtype, a); }

bool conv_img_ok(int dtype, const ConvArgs &a) {
  return dtype == GCPSL_BF16 && a.taps == 9 && a.H == IMG && a.W == IMG && (a.Csrc == 32 || a.Csrc == 64) &&
         (a.N == 32 || a.N == 64) && !(a.Csrc == 64 && a.N == 64) && a.res == nullptr &&
         a.Kp == ((9 * a.Csrc + 63) / 64) * 64;
}

// Every instantiation is named in this (non-template) function.
hipError_t launch_conv_img(const ConvArgs &a, hipStream_t s, std::string *label) {
  if (!conv_img_ok(GCPSL_BF16, a)) return hipErrorInvalidValue;
  // the forward of a 32-channel input takes two image rows per wave (16-row
  // tiles, so the weight matrix is staged once per 512 pixels); a 64-channel
  // input's 18-row halo would not leave room for two workgroups per CU
  const int rpw = (a.epi == EPI_FWD && a.Csrc == 32) ? 2 : 1;
  const int MT = a.Bt * IMG / (8 * rpw);  // tiles of 8 rpw image rows per replica
  const dim3 g((uint32_t)MT * a.C);
  if (label)
    *label = std::string(a.epi == EPI_FWD ? "conv_fwd" : "conv_dgrad") + "<bf16," + std::to_string(256 * rpw) +
             "x" + std::to_string(a.N) + "x" + std::to_string(9 * a.Csrc) + ",w8,img>";
#define IMG_GO(CS, NO, E, RPW) \
  hipLaunchKernelGGL((conv_img_kernel<CS, NO, E, RPW>), g, dim3(NTHR), (ImgCfg<CS, NO, RPW>::LDS), s, a, MT)
  static_assert(ImgCfg<32, 32, 2>::FITS2 && ImgCfg<32, 64, 2>::FITS2 && ImgCfg<32, 32>::FITS2 &&
                    ImgCfg<32, 64>::FITS2 && ImgCfg<64, 32>::FITS2,
                "two per CU");
  static PerDeviceOnce attr;
  if (attr.needed()) {
    for (const void *f : {reinterpret_cast<const void *>(&conv_img_kernel<64, 32, EPI_FWD, 1>),
                          reinterpret_cast<const void *>(&conv_img_kernel<64, 32, EPI_DGRAD, 1>)}) {
      const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, ImgCfg<64, 32>::LDS);
      if (e != hipSuccess) return e;
    }
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&conv_img_kernel<32, 64, EPI_FWD, 2>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, ImgCfg<32, 64, 2>::LDS);
    if (e != hipSuccess) return e;
    attr.mark();
  }
  if (a.epi == EPI_FWD) {
    if (a.Csrc == 32 && a.N == 32) IMG_GO(32, 32, EPI_FWD, 2);
    else if (a.Csrc == 32) IMG_GO(32, 64, EPI_FWD, 2);
    else IMG_GO(64, 32, EPI_FWD, 1);
  } else {
    if (a.Csrc == 32 && a.N == 32) IMG_GO(32, 32, EPI_DGRAD, 1);
    else if (a.Csrc == 32) IMG_GO(32, 64, EPI_DGRAD, 1);
    else IMG_GO(64, 32, EPI_DGRAD, 1);
  }
#undef IMG_GO
  return hipGetLastError();
}
