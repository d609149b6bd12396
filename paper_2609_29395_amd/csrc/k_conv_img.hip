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

// The forward of a 32-channel input followed by the 2 x 2 max pool with
// routing codes (the client's last conv before the cut), persistent: one
// workgroup of 16 waves per CU; workgroup w of replica slot z takes the
// 16-row tiles w, w + WPR, w + 2 WPR, ... of its replica, alternately by its
// two teams of 8 waves.  The weight matrix is copied into LDS once per
// workgroup and shared by both teams; each team has its own halo buffer.
// While one team runs a tile's MFMAs, the other copies its next halo and
// pools and stores its previous tile (127 KB of LDS with the bias and the
// copy table, at most 128 registers per wave; a third halo buffer, so that
// a copy could start a phase earlier, measured slower).
// Pixel fragment tm = 2 rr + hf of a wave holds the columns 2 li + hf of its
// image row rr, so a lane ends with whole 2 x 2 pooling windows (4 channels
// of pooled column li) and pools them in registers.  A halo row keeps its
// even columns, then its odd ones (column w' in slot (w' mod 2) 17 + w' / 2),
// and slot i keeps its 16-byte chunk c at c ^ ((i >> 1) & 3), so that the
// 16-byte reads of 8 consecutive lanes (consecutive slots of one half) fall
// on distinct banks; weight rows are 656 bytes apart (40 chunks and one of
// padding) for the same reason, and a tap's fragments sit a fixed 64 bytes
// after the previous tap's.
template <int N> __device__ __forceinline__ void img_wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// packed 16-bit integer arithmetic (two halves per register), kept as such
// (the compiler would otherwise split min(x, 1) into compares, and it has
// folded a packed signed maximum of the second word of a loaded pair onto
// the first word's)
__device__ __forceinline__ uint32_t pk_max_i16(uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_pk_max_i16 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ uint32_t pk_max0_i16(uint32_t a) {
  uint32_t r;
  asm("v_pk_max_i16 %0, %1, 0" : "=v"(r) : "v"(a));
  return r;
}
__device__ __forceinline__ uint32_t pk_sub_u16(uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_pk_sub_u16 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ uint32_t pk_min_u16(uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_pk_min_u16 %0, %1, %2" : "=v"(r) : "v"(a), "s"(b));
  return r;
}
__device__ __forceinline__ uint32_t pk_add_u16(uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_pk_add_u16 %0, %1, %2" : "=v"(r) : "v"(a), "s"(b));
  return r;
}
__device__ __forceinline__ uint32_t pk_mad_u16(uint32_t a, uint32_t b, uint32_t c) {
  uint32_t r;
  asm("v_pk_mad_u16 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "s"(c));
  return r;
}
__device__ __forceinline__ uint32_t pk_mul_lo_u16(uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_pk_mul_lo_u16 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// the lane's index within its wave, computed afresh (mbcnt over all lanes)
__device__ __forceinline__ int img_lane_id() {
  int v;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(v));
  return v;
}

template <int OFF> __device__ __forceinline__ void lds_read16(u32x4 &v, uint32_t ad) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset");
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(ad), "n"(OFF));
}

constexpr int IMGP_WROW = 656;  // bytes per weight row in LDS: 40 chunks and one of padding

template <int TAP, int TN, int TN0 = 0> __device__ __forceinline__ void img_pool_wfrags(u32x4 (&w)[TN], uint32_t wb) {
  if constexpr (TN0 < TN) {
    // fragment tn: 16 weight rows further
    lds_read16<64 * TAP + TN0 * 16 * IMGP_WROW>(w[TN0], wb);
    img_pool_wfrags<TAP, TN, TN0 + 1>(w, wb);
  }
}

// tap (r, s) = (TAP / 3, TAP % 3) of a 16-row tile: weight fragment tn at
// wb + tn 16 rows + 64 TAP, pixel fragment tm = 2 rr + hf (columns
// 2 li + hf + s) at xb[hf + s] + (rr + r) halo rows
template <int TAP, int TN>
__device__ __forceinline__ void img_pool_tap(f32x4_t (&acc)[4][TN], uint32_t wb, const uint32_t (&xb)[4]) {
  constexpr int r = TAP / 3, s = TAP % 3, ROWB = HP * 64;  // bytes per halo row of 32 channels
  u32x4 w[TN], x[4];
  img_pool_wfrags<TAP, TN>(w, wb);
  lds_read16<r * ROWB>(x[0], xb[s]);
  lds_read16<r * ROWB>(x[1], xb[s + 1]);
  lds_read16<(r + 1) * ROWB>(x[2], xb[s]);
  lds_read16<(r + 1) * ROWB>(x[3], xb[s + 1]);
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int i = 0; i < TN; ++i) asm volatile("" : "+v"(w[i]));
#pragma unroll
  for (int i = 0; i < 4; ++i) asm volatile("" : "+v"(x[i]));
#pragma unroll
  for (int tm = 0; tm < 4; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) mma(acc[tm][tn], w[tn], x[tm]);
}

// LDS of the ping-pong kernel: two halo buffers, the weights, the bias
template <int NO> struct ImgPool {
  using CF = ImgCfg<32, NO, 2>;
  // padded weight rows, in whole 1 KB copies (so that no copy reaches the bias)
  static constexpr int W_LDS = (NO * IMGP_WROW + 1023) / 1024 * 1024;
  static constexpr int W_OFF = 2 * CF::H_BYTES, B_OFF = W_OFF + W_LDS;
  // the bias (256 bytes), then each team thread's halo copy table (16 bytes)
  static constexpr int T_OFF = B_OFF + 256, LDS = T_OFF + NTHR * 16;
  static_assert(NO * 4 <= 256 && CF::HQ <= 8, "bias and table sizes");
  static_assert(LDS <= 160 * 1024, "one workgroup per CU");
};

template <int NO>
__global__ void __launch_bounds__(2 * NTHR)
conv_img_pool_kernel(ConvArgs a, int MT, int WPR) {
  using CF = ImgCfg<32, NO, 2>;
  using PL = ImgPool<NO>;
  constexpr int CS = 32, TROWS = CF::TROWS, HPIX = CF::HPIX, TN = CF::TN, CPR = CF::CPR;
  constexpr int W_OFF = PL::W_OFF, B_OFF = PL::B_OFF, T_OFF = PL::T_OFF;
  constexpr int NST = 2 * TN;  // global stores per wave and tile (pooled values and codes per fragment)
  static_assert(CPR == 4 && CF::KP * 2 == 640 && HP == 34, "4 chunks per halo pixel, 640-byte weight rows");
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int team = wave >> 3, tw = wave & 7;  // team 0 takes the even tiles, team 1 the odd ones
  const uint32_t t = xcd_swizzle(blockIdx.x, (uint32_t)(WPR * a.C));
  const int z = __builtin_amdgcn_readfirstlane((int)(t / (uint32_t)WPR));
  const int w0 = __builtin_amdgcn_readfirstlane((int)(t - (uint32_t)z * (uint32_t)WPR));
  const int nt = (MT - w0 + WPR - 1) / WPR;  // tiles of this workgroup: w0 + k WPR, k < nt
  const int rep = replica_of(a.rmap, z);
  const int M = a.Bt * IMG * IMG;
  const bf16_t *src = reinterpret_cast<const bf16_t *>(a.src) + rep * a.src_rs;
  const bf16_t *wt = reinterpret_cast<const bf16_t *>(a.wt) + rep * a.wt_rs;
  const __amdgpu_buffer_rsrc_t rss = rsrc(src, (uint32_t)((int64_t)M * CS * 2));
  const __amdgpu_buffer_rsrc_t rsw = rsrc(wt, (uint32_t)CF::W_BYTES);

  // the weight matrix, once, by all 16 waves: row n at n * 656 bytes, its
  // 40 chunks in order and a zero one
  constexpr int WSLOTS = PL::W_LDS / 16, WROWC = IMGP_WROW / 16;
#pragma unroll
  for (int q = 0; q < (WSLOTS + 2 * NTHR - 1) / (2 * NTHR); ++q) {
    const int slot0 = q * 2 * NTHR + wave * 64;
    if (slot0 < WSLOTS) {  // (whole 64-slot copies: WSLOTS is a multiple of 64)
      const int j = slot0 + lane;
      const int row = j / WROWC, kc = j % WROWC;
      const uint32_t off = (row < NO && kc < CF::WCH) ? (uint32_t)(row * CF::KP + 8 * kc) * 2u : kOob;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsw, LDS_PTR(smem + W_OFF + slot0 * 16), 16, off, 0, 0, 0);
    }
  }
  // The halo image rows h0 - 1 .. h0 + 16 of tile k with a one-pixel zero
  // border, copied by the 8 waves of its team into the team's buffer.  A
  // thread's 16-byte piece q lands in the same halo slot for every tile, so
  // its source is tabled once per thread (ent, 16 bits per piece): the
  // offset from the tile's first pixel in 16-byte units plus 128, and flags
  // for a slot outside the image in the upper tile of an image (0x8000: the
  // row above it), in the lower one (0x4000: the row below) and always
  // (0x2000: the border columns, the padding past the halo).
  auto issue_halo = [&](int k, const u32x4 &ent) {
    const int m0 = (w0 + k * WPR) * (TROWS * IMG), h0 = (m0 / IMG) % IMG;
    const uint32_t bad = h0 == 0 ? 0xa000u : 0x6000u;
    const uint32_t base = (uint32_t)m0 * (CS * 2) - 128u * 16u;
#pragma unroll
    for (int q = 0; q < CF::HQ; ++q) {
      const int byte = q * NTHR * 16 + tw * 1024;
      if (byte < CF::H_BYTES) {
        const uint32_t e = (ent[q >> 1] >> (16 * (q & 1))) & 0xffffu;
        const uint32_t off = (e & bad) ? kOob : base + (e & 0x1fffu) * 16u;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rss, LDS_PTR(smem + team * CF::H_BYTES + byte), 16, off, 0, 0, 0);
      }
    }
  };
  if (team == 0) {
    // the table: slot R of a halo row is column w' = 2 (R mod 17) + R / 17
    // (even columns, then odd ones), and chunk c sits at c ^ ((w' >> 2) & 3)
    uint32_t e16[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) e16[q] = 0x2000u;
#pragma unroll
    for (int q = 0; q < CF::HQ; ++q) {
      const int j = q * NTHR + tw * 64 + lane;
      const int R = j / CPR, cs = j % CPR;
      const int hp = R / HP, rem = R - hp * HP;
      const int idx = rem % (HP / 2), wp = 2 * idx + rem / (HP / 2);
      const int c = cs ^ ((idx >> 1) & (CPR - 1));
      const int w = wp - 1;
      if (R < HPIX && (unsigned)w < (unsigned)IMG)
        e16[q] = (uint32_t)(((hp - 1) * IMG + w) * CPR + c + 128) | (hp == 0 ? 0x8000u : 0u) |
                 (hp == HPIX / HP - 1 ? 0x4000u : 0u);
    }
    const u32x4 ent = {e16[0] | (e16[1] << 16), e16[2] | (e16[3] << 16), e16[4] | (e16[5] << 16),
                       e16[6] | (e16[7] << 16)};
    *reinterpret_cast<u32x4 *>(smem + T_OFF + (tw * 64 + lane) * 16) = ent;
    issue_halo(0, ent);
  }
  // the bias into LDS (read back with LDS reads the compiler does not see,
  // so that it adds no wait for the copies in flight); loaded after the
  // copies, so waiting for it also waits for them
  if (tid < NO) reinterpret_cast<float *>(smem + B_OFF)[tid] = a.bias[rep * a.bias_rs + tid];
  img_wait_vm<0>();
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");

  const uint32_t lds0 = (uint32_t)(size_t)LDS_PTR(smem);
  bf16_t *zo = reinterpret_cast<bf16_t *>(a.pool_out) + rep * a.pool_rs;
  uint8_t *co = a.pool_code + rep * a.pool_rs;

  // Phase ph: the team of tile ph (ph & 1) computes it from its buffer; the
  // other team first copies its next tile (ph + 1) into its own buffer (read
  // for the last time in phase ph - 1), then pools and stores its tile
  // ph - 1, then waits for its copies.  One barrier per phase, so a copy has
  // the other team's whole k loop to land, and the pooling of one team runs
  // beside the other team's MFMAs.
  f32x4_t acc[4][TN];
  for (int ph = 0; ph <= nt; ++ph) {
    if ((ph & 1) == team) {
      if (ph < nt) {
        // the accumulators start from the bias of their channels tn*16 +
        // 4 lg .. + 3 (read with its own wait)
        const uint32_t ba = lds0 + (uint32_t)(B_OFF + 16 * (img_lane_id() >> 4));
        f32x4_t bv[4];
        if constexpr (TN == 4)
          asm volatile(
              "ds_read_b128 %0, %4 offset:0\n\tds_read_b128 %1, %4 offset:64\n\t"
              "ds_read_b128 %2, %4 offset:128\n\tds_read_b128 %3, %4 offset:192\n\ts_waitcnt lgkmcnt(0)"
              : "=&v"(bv[0]), "=&v"(bv[1]), "=&v"(bv[2]), "=&v"(bv[3])
              : "v"(ba)
              : "memory");
        else
          asm volatile("ds_read_b128 %0, %2 offset:0\n\tds_read_b128 %1, %2 offset:64\n\ts_waitcnt lgkmcnt(0)"
                       : "=&v"(bv[0]), "=&v"(bv[1])
                       : "v"(ba)
                       : "memory");
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[i][tn] = bv[tn];
        // fragment read bases (from an opaque lane index, so that they are
        // not held across the pooling branch): weight row li, chunk lg of
        // tap 0; the team's halo buffer, pixel 2 li + hf + s of the wave's
        // first halo row, chunk lg
        const int ln = img_lane_id();
        const int li = ln & 15, lg = ln >> 4;
        const uint32_t wb = lds0 + (uint32_t)(W_OFF + li * IMGP_WROW + lg * 16);
        const uint32_t hb = lds0 + (uint32_t)(team * CF::H_BYTES + 2 * tw * HP * CF::RB);
        uint32_t xk[4];  // columns 2 li + e: plane e & 1, slot li + e / 2 of it
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int idx = li + (e >> 1);
          xk[e] = hb + (uint32_t)(((e & 1) * (HP / 2) + idx) * CF::RB + ((lg ^ ((idx >> 1) & (CPR - 1))) * 16));
        }
        img_pool_tap<0>(acc, wb, xk);
        img_pool_tap<1>(acc, wb, xk);
        img_pool_tap<2>(acc, wb, xk);
        img_pool_tap<3>(acc, wb, xk);
        img_pool_tap<4>(acc, wb, xk);
        img_pool_tap<5>(acc, wb, xk);
        img_pool_tap<6>(acc, wb, xk);
        img_pool_tap<7>(acc, wb, xk);
        img_pool_tap<8>(acc, wb, xk);
      }
    } else {
      if (ph + 1 < nt) {
        u32x4 ent;
        const uint32_t ta = lds0 + (uint32_t)(T_OFF + (tw * 64 + img_lane_id()) * 16);
        asm volatile("ds_read_b128 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(ent) : "v"(ta) : "memory");
        issue_halo(ph + 1, ent);
      }
      if (ph >= 1) {
        // pooling: lane (li, lg) holds channels tn*16 + 4 lg + e of columns
        // 2 li (hf 0) and 2 li + 1 (hf 1) of image rows 2 tw (rr 0) and
        // 2 tw + 1 (rr 1) -- pooled pixel li of pooled row h0 / 2 + tw.  The
        // pre-activations are rounded to bf16 as the unpooled layer would
        // store them (ReLU commutes with the rounding).  Positive bf16 values
        // order as their bits read as signed 16-bit integers, and every
        // other value (negative, -0) reads as at most 0, so the window's
        // maximum with 0 is the pooled ReLU output, taken two channels at a
        // time by packed 16-bit integer operations; the code is the first
        // window position (row-major) holding it, or 4 where it is 0.
        // (Lane-derived addresses from an opaque lane index, not held
        // across the k loop.)
        const int ln = img_lane_id();
        const int eli = ln & 15, elg = ln >> 4;
        const int m0 = (w0 + (ph - 1) * WPR) * (TROWS * IMG);
        const int b = m0 / (IMG * IMG), hz = ((m0 / IMG) % IMG) / 2 + tw;
        const int64_t zrow = ((int64_t)(b * (IMG / 2) + hz) * (IMG / 2) + eli) * NO + 4 * elg;
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          uint32_t zz[2], cc[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            // channels 2h, 2h + 1 of the four window positions p = 2 rr + hf
            uint32_t v[4];
#pragma unroll
            for (int p = 0; p < 4; ++p) v[p] = pack2_bf16(acc[p][tn][2 * h], acc[p][tn][2 * h + 1]);
            const uint32_t m = pk_max0_i16(pk_max_i16(pk_max_i16(v[0], v[1]), pk_max_i16(v[2], v[3])));
            // ne_p = min(m - v_p, 1) is 0 exactly where position p holds the
            // maximum (m >= v_p, so the 16-bit difference is m - v_p); the
            // first such p is ne_0 (1 + ne_1 (1 + ne_2)) (3 when none of
            // 0..2 does), and 4 replaces it where the maximum is 0
            const uint32_t one = 0x00010001u, four = 0x00040004u;
            const uint32_t mb = m;
            uint32_t ne[3];
#pragma unroll
            for (int p = 0; p < 3; ++p) ne[p] = pk_min_u16(pk_sub_u16(mb, v[p]), one);
            const uint32_t first = pk_mul_lo_u16(ne[0], pk_mad_u16(ne[1], pk_add_u16(ne[2], one), one));
            const uint32_t pos = pk_min_u16(mb, one);
            zz[h] = mb;
            cc[h] = pk_mad_u16(pk_sub_u16(first, four), pos, four);
          }
          // codes of channels 0..3: the low bytes of the four 16-bit codes
          const uint32_t code = __builtin_amdgcn_perm(cc[1], cc[0], 0x06040200u);
          *reinterpret_cast<u32x2 *>(zo + zrow + tn * 16) = u32x2{zz[0], zz[1]};
          *reinterpret_cast<uint32_t *>(co + zrow + tn * 16) = code;
        }
        // this team's copies have landed (they were issued before the NST
        // stores, and the vector memory counter retires in issue order)
        img_wait_vm<NST>();
      } else {
        img_wait_vm<0>();
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  }
}

// The input gradient of the cut layer (64 gradient channels at the pooled
// resolution, 32 input channels), persistent and ping-ponged like the
// forward above: one workgroup of 16 waves per CU walks every WPR-th 8-row
// tile of one replica, alternately by its two teams of 8 waves (one image
// row per wave).  The weight matrix is copied into LDS once per workgroup;
// each team has its own halo buffer, which it fills for its next tile while
// the other team runs its MFMAs: it loads the pooled gradient and the
// routing codes of each halo piece into registers, then masks and stores its
// previous tile, then writes the pieces routed (the gradient where the code
// names the pixel's window position, zero elsewhere).  Each thread's pieces
// sit at fixed halo slots, so their sources are tabled once in LDS.  A halo
// pixel row is 128 bytes with chunk c at c ^ (w' & 7), weight rows are 1168
// bytes apart (72 chunks and one of padding): the 16-byte fragment reads of
// 8 consecutive lanes fall on distinct banks.
constexpr int IMGD_WROW = 1168;  // bytes per weight row in LDS: 72 chunks and one of padding

// tap (r, s) = (TAP / 3, TAP % 3): both 32-channel k groups; weight fragment
// (tn, g) at wb + tn 16 rows + TAP 128 + g 64 bytes, pixel fragment (half, g)
// at xb[s][g] + r halo rows + half 16 pixels
template <int TAP>
__device__ __forceinline__ void img_dgrad_tap(f32x4_t (&acc)[2][2], uint32_t wb, const uint32_t (&xb)[3][2]) {
  constexpr int r = TAP / 3, s = TAP % 3, ROWB = HP * 128;
  u32x4 w[2][2], x[2][2];  // [g][tn], [g][half]
  lds_read16<TAP * 128>(w[0][0], wb);
  lds_read16<16 * IMGD_WROW + TAP * 128>(w[0][1], wb);
  lds_read16<TAP * 128 + 64>(w[1][0], wb);
  lds_read16<16 * IMGD_WROW + TAP * 128 + 64>(w[1][1], wb);
  lds_read16<r * ROWB>(x[0][0], xb[s][0]);
  lds_read16<r * ROWB + 16 * 128>(x[0][1], xb[s][0]);
  lds_read16<r * ROWB>(x[1][0], xb[s][1]);
  lds_read16<r * ROWB + 16 * 128>(x[1][1], xb[s][1]);
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int g = 0; g < 2; ++g)
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      asm volatile("" : "+v"(w[g][i]));
      asm volatile("" : "+v"(x[g][i]));
    }
#pragma unroll
  for (int g = 0; g < 2; ++g)
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int tn = 0; tn < 2; ++tn) mma(acc[hf][tn], w[g][tn], x[g][hf]);
}

// LDS of the input-gradient kernel: two halo buffers, the weights, the table
struct ImgDgrad {
  using CF = ImgCfg<64, 32, 1>;
  static constexpr int W_LDS = (32 * IMGD_WROW + 1023) / 1024 * 1024;
  static constexpr int W_OFF = 2 * CF::H_BYTES, T_OFF = W_OFF + W_LDS, LDS = T_OFF + NTHR * 16;
  static_assert(CF::HQ <= 8 && CF::TROWS == 8 && CF::CPR == 8 && CF::KP == 576, "8-row tiles of 64 channels");
  static_assert(LDS <= 160 * 1024, "one workgroup per CU");
};

__global__ void __launch_bounds__(2 * NTHR)
conv_img_dgrad_kernel(ConvArgs a, int MT, int WPR) {
  using CF = ImgCfg<64, 32, 1>;
  using PL = ImgDgrad;
  constexpr int CS = 64, NO = 32, TROWS = 8, HPIX = CF::HPIX, CPR = CF::CPR, HQ = CF::HQ;
  constexpr int W_OFF = PL::W_OFF, T_OFF = PL::T_OFF;
  constexpr int PW = IMG / 2;  // pooled side
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int team = wave >> 3, tw = wave & 7;  // team 0 takes the even tiles, team 1 the odd ones
  const uint32_t t = xcd_swizzle(blockIdx.x, (uint32_t)(WPR * a.C));
  const int z = __builtin_amdgcn_readfirstlane((int)(t / (uint32_t)WPR));
  const int w0 = __builtin_amdgcn_readfirstlane((int)(t - (uint32_t)z * (uint32_t)WPR));
  const int nt = (MT - w0 + WPR - 1) / WPR;  // tiles of this workgroup: w0 + k WPR, k < nt
  const int rep = replica_of(a.rmap, z);
  const bf16_t *gsrc = reinterpret_cast<const bf16_t *>(a.src) + rep * a.src_rs;  // pooled gradient
  const uint8_t *csrc = a.pool_code + rep * a.src_rs;                              // its codes
  const bf16_t *wt = reinterpret_cast<const bf16_t *>(a.wt) + rep * a.wt_rs;
  const bf16_t *msk = reinterpret_cast<const bf16_t *>(a.mask) + rep * a.out_rs;
  bf16_t *out = reinterpret_cast<bf16_t *>(a.out) + rep * a.out_rs;
  const __amdgpu_buffer_rsrc_t rsw = rsrc(wt, (uint32_t)CF::W_BYTES);

  // the weight matrix, once, by all 16 waves: row n at n * 1168 bytes, its
  // 72 chunks in order and a zero one
  constexpr int WSLOTS = PL::W_LDS / 16, WROWC = IMGD_WROW / 16;
#pragma unroll
  for (int q = 0; q < (WSLOTS + 2 * NTHR - 1) / (2 * NTHR); ++q) {
    const int slot0 = q * 2 * NTHR + wave * 64;
    if (slot0 < WSLOTS) {  // (whole 64-slot copies: WSLOTS is a multiple of 64)
      const int j = slot0 + lane;
      const int row = j / WROWC, kc = j % WROWC;
      const uint32_t off = (row < NO && kc < CF::WCH) ? (uint32_t)(row * CF::KP + 8 * kc) * 2u : kOob;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsw, LDS_PTR(smem + W_OFF + slot0 * 16), 16, off, 0, 0, 0);
    }
  }

  // A thread's halo piece q of a tile (16-byte slot j = 512 q + 64 tw + lane
  // of its team's buffer: pixel slot j / 8, chunk j % 8) is tabled as 16 bits:
  // the pooled piece it comes from, counted in 16-byte units from the tile's
  // pooled row above (10 bits), the pixel's window position (2 bits), and
  // flags for a pixel outside the image in the top tile of an image (0x8000:
  // the row above it), in the bottom tile (0x4000: the row below) and always
  // (0x2000: the border columns, the padding past the halo).
  u32x4 ent0;
  if (team == 0) {
    uint32_t e16[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) e16[q] = 0x2000u;
#pragma unroll
    for (int q = 0; q < HQ; ++q) {
      const int j = q * NTHR + tw * 64 + lane;
      const int R = j / CPR, cs = j % CPR;
      const int hp = R / HP, wp = R - hp * HP;
      const int c = cs ^ (wp & 7);
      const int w = wp - 1;
      if (R < HPIX && (unsigned)w < (unsigned)IMG) {
        const int prr = (hp + 1) >> 1;  // pooled row of image row h0 - 1 + hp, from the one above h0 / 2
        const int pos = (((hp - 1) & 1) << 1) | (w & 1);
        e16[q] = (uint32_t)((prr * PW + (w >> 1)) * CPR + c) | ((uint32_t)pos << 10) | (hp == 0 ? 0x8000u : 0u) |
                 (hp == HPIX / HP - 1 ? 0x4000u : 0u);
      }
    }
    ent0 = u32x4{e16[0] | (e16[1] << 16), e16[2] | (e16[3] << 16), e16[4] | (e16[5] << 16), e16[6] | (e16[7] << 16)};
    *reinterpret_cast<u32x4 *>(smem + T_OFF + (tw * 64 + lane) * 16) = ent0;
  }
  // the pooled gradient and codes of this thread's pieces of tile k, into
  // registers (every load is issued, from a valid address; the flags are
  // applied when the pieces are routed)
  u32x4 gv[HQ];
  u32x2 cv[HQ];
  auto load_halo = [&](int k, const u32x4 &ent) {
    const int m0 = (w0 + k * WPR) * (TROWS * IMG), h0 = (m0 / IMG) % IMG;
    const int pbase = ((m0 / (IMG * IMG)) * PW * PW + (h0 / 2 - 1) * PW) * CS;  // element of the pooled row above
    // a piece outside the image (above the first or below the last pooled
    // row too) reads the replica's first piece instead
    const uint32_t bad = h0 == 0 ? 0xa000u : (h0 == IMG - TROWS ? 0x6000u : 0x2000u);
#pragma unroll
    for (int q = 0; q < HQ; ++q) {
      if (q * NTHR * 16 + tw * 1024 < CF::H_BYTES) {
        const uint32_t e = (ent[q >> 1] >> (16 * (q & 1))) & 0xffffu;
        const int el = (e & bad) ? 0 : pbase + (int)(e & 0x3ffu) * 8;
        gv[q] = *reinterpret_cast<const u32x4 *>(gsrc + el);
        cv[q] = *reinterpret_cast<const u32x2 *>(csrc + el);
      }
    }
  };
  // the routed pieces into the team's halo buffer
  auto route_halo = [&](int k, const u32x4 &ent) {
    const int m0 = (w0 + k * WPR) * (TROWS * IMG), h0 = (m0 / IMG) % IMG;
    const uint32_t bad = h0 == 0 ? 0xa000u : (h0 == IMG - TROWS ? 0x6000u : 0x2000u);
    const int ln = img_lane_id();
#pragma unroll
    for (int q = 0; q < HQ; ++q) {
      const int byte = q * NTHR * 16 + tw * 1024;
      if (byte < CF::H_BYTES) {
        const uint32_t e = (ent[q >> 1] >> (16 * (q & 1))) & 0xffffu;
        const uint32_t kpos = (e & bad) ? 0xffu : (e >> 10) & 3u;  // 0xff: no code matches
        u32x4 v;
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          const uint32_t cb = cv[q][d >> 1] >> (16 * (d & 1));  // codes of channels 2d, 2d + 1
          const uint32_t keep = ((cb & 0xffu) == kpos ? 0x0000ffffu : 0u) | (((cb >> 8) & 0xffu) == kpos ? 0xffff0000u : 0u);
          v[d] = gv[q][d] & keep;
        }
        const uint32_t ad = (uint32_t)(size_t)LDS_PTR(smem + team * CF::H_BYTES + byte) + (uint32_t)ln * 16u;
        asm volatile("ds_write_b128 %0, %1" ::"v"(ad), "v"(v) : "memory");
      }
    }
  };
  if (team == 0) {
    load_halo(0, ent0);
    img_wait_vm<0>();
    route_halo(0, ent0);
  }
  img_wait_vm<0>();
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");

  const uint32_t lds0 = (uint32_t)(size_t)LDS_PTR(smem);
  // Phase ph: the team of tile ph (ph & 1) computes it from its buffer; the
  // other team loads its next tile's pieces (ph + 1), masks and stores its
  // tile ph - 1, then routes the pieces into its buffer (read for the last
  // time in phase ph - 1).  One barrier per phase.
  f32x4_t acc[2][2];
  for (int ph = 0; ph <= nt; ++ph) {
    if ((ph & 1) == team) {
      if (ph < nt) {
        // fragment read bases (from an opaque lane index): weight row li,
        // chunk lg; the team's halo buffer, pixel li + s of the wave's first
        // halo row, chunk 4 g + lg
        const int ln = img_lane_id();
        const int li = ln & 15, lg = ln >> 4;
        const uint32_t wb = lds0 + (uint32_t)(W_OFF + li * IMGD_WROW + lg * 16);
        uint32_t xb[3][2];
#pragma unroll
        for (int s = 0; s < 3; ++s)
#pragma unroll
          for (int g = 0; g < 2; ++g)
            xb[s][g] = lds0 + (uint32_t)(team * CF::H_BYTES + (tw * HP + li + s) * CF::RB +
                                         (((4 * g + lg) ^ ((li + s) & 7)) * 16));
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int k = 0; k < 2; ++k) acc[i][k] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        img_dgrad_tap<0>(acc, wb, xb);
        img_dgrad_tap<1>(acc, wb, xb);
        img_dgrad_tap<2>(acc, wb, xb);
        img_dgrad_tap<3>(acc, wb, xb);
        img_dgrad_tap<4>(acc, wb, xb);
        img_dgrad_tap<5>(acc, wb, xb);
        img_dgrad_tap<6>(acc, wb, xb);
        img_dgrad_tap<7>(acc, wb, xb);
        img_dgrad_tap<8>(acc, wb, xb);
      }
    } else {
      const bool next = ph + 1 < nt;
      u32x4 ent;
      if (next) {
        const uint32_t ta = lds0 + (uint32_t)(T_OFF + (tw * 64 + img_lane_id()) * 16);
        asm volatile("ds_read_b128 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(ent) : "v"(ta) : "memory");
      }
      if (ph >= 1) {
        // lane (li, lg) holds channels tn*16 + 4 lg + e of pixel
        // 16 half + li of image row h0 + tw; the gradient passes where the
        // layer below's output (the mask) is positive (positive bf16 values
        // read as positive 16-bit integers)
        const int ln = img_lane_id();
        const int eli = ln & 15, elg = ln >> 4;
        const int64_t p0 = (int64_t)(w0 + (ph - 1) * WPR) * (TROWS * IMG) + tw * IMG + eli;
        u32x2 mv[2][2];
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int tn = 0; tn < 2; ++tn)
            mv[hf][tn] = *reinterpret_cast<const u32x2 *>(msk + (p0 + 16 * hf) * NO + tn * 16 + 4 * elg);
        if (next) load_halo(ph + 1, ent);
        if (next) img_wait_vm<2 * HQ>();  // the masks (issued before the pieces)
        else img_wait_vm<0>();
        const uint32_t one = 0x00010001u;
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int tn = 0; tn < 2; ++tn) {
            u32x2 o;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              const uint32_t v = pack2_bf16(acc[hf][tn][2 * h], acc[hf][tn][2 * h + 1]);
              // 1 where the mask is positive, else 0, per 16-bit half
              const uint32_t pass = pk_min_u16(pk_max0_i16(mv[hf][tn][h]), one);
              o[h] = pk_mul_lo_u16(v, pass);
            }
            *reinterpret_cast<u32x2 *>(out + (p0 + 16 * hf) * NO + tn * 16 + 4 * elg) = o;
          }
        if (next) img_wait_vm<4>();  // the pieces (issued before the 4 stores)
      } else if (next) {
        load_halo(ph + 1, ent);
        img_wait_vm<0>();
      }
      if (next) route_halo(ph + 1, ent);
    }
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
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
  // the forward into the pool and its codes: persistent workgroups, one per
  // CU, each taking every WPR-th tile of its replica
  const bool pers = a.epi == EPI_FWD && a.Csrc == 32 && a.pool_out && a.pool_code && !a.no_relu;
  // the input gradient from the pooled gradient and its codes, with a mask:
  // persistent the same way
  const bool pdg = a.epi == EPI_DGRAD && a.Csrc == 64 && a.N == 32 && a.pool_code && a.mask;
  if (label)
    *label = std::string(a.epi == EPI_FWD ? "conv_fwd" : "conv_dgrad") + "<bf16," + std::to_string(256 * rpw) +
             "x" + std::to_string(a.N) + "x" + std::to_string(9 * a.Csrc) +
             (pers || pdg ? ",w8,img,pool>" : ",w8,img>");
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
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&conv_img_kernel<32, 64, EPI_FWD, 2>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, ImgCfg<32, 64, 2>::LDS);
    if (e != hipSuccess) return e;
    e = hipFuncSetAttribute(reinterpret_cast<const void *>(&conv_img_dgrad_kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, ImgDgrad::LDS);
    if (e != hipSuccess) return e;
    for (const void *f : {reinterpret_cast<const void *>(&conv_img_pool_kernel<64>),
                          reinterpret_cast<const void *>(&conv_img_pool_kernel<32>)}) {
      e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize,
                              f == reinterpret_cast<const void *>(&conv_img_pool_kernel<64>) ? ImgPool<64>::LDS
                                                                                             : ImgPool<32>::LDS);
      if (e != hipSuccess) return e;
    }
    attr.mark();
  }
  if (pers) {
    constexpr int kSlots = 256;  // one workgroup on each of the 256 CUs
    const int want = std::max(1, std::min(MT, kSlots / std::max(1, a.C)));
    const int per = (MT + want - 1) / want;  // tiles per workgroup
    const int wpr = (MT + per - 1) / per;
    const dim3 gp((uint32_t)wpr * a.C);
    if (a.N == 64)
      hipLaunchKernelGGL(conv_img_pool_kernel<64>, gp, dim3(2 * NTHR), ImgPool<64>::LDS, s, a, MT, wpr);
    else
      hipLaunchKernelGGL(conv_img_pool_kernel<32>, gp, dim3(2 * NTHR), ImgPool<32>::LDS, s, a, MT, wpr);
    return hipGetLastError();
  }
  if (pdg) {
    constexpr int kSlots = 256;
    const int want = std::max(1, std::min(MT, kSlots / std::max(1, a.C)));
    const int per = (MT + want - 1) / want;
    const int wpr = (MT + per - 1) / per;
    hipLaunchKernelGGL(conv_img_dgrad_kernel, dim3((uint32_t)wpr * a.C), dim3(2 * NTHR), ImgDgrad::LDS, s, a, MT, wpr);
    return hipGetLastError();
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
