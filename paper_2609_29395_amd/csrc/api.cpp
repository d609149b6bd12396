// Host runtime of the C ABI: model plan, workspace layout and the order of
// kernel launches for sampling, one local round, fusion and participation.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "runtime.h"

// ------------------------------------------------------------------ errors
namespace {
thread_local std::string g_err;
}
void gcpsl_clear_error() { g_err.clear(); }
int gcpsl_fail(int code, const std::string &msg) {
  g_err = msg;
  return code;
}
extern "C" const char *gcpsl_last_error(void) { return g_err.c_str(); }

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
int round_up(int x, int m) { return (x + m - 1) / m * m; }

// Pixels per chunk of a channel reduction over px pixels of each of C
// replicas: halved from 256 down to 16 until there are about 2048 chunks in
// all, so that small late-stage tensors still spread over the chip.
int norm_chunk(int64_t px, int C) {
  int ch = 256;
  while (ch > 16 && (px + ch - 1) / ch * C < 2048) ch >>= 1;
  return ch;
}

struct LayerInfo {
  gcpsl_layer spec{};
  int H = 0, W = 0, Ci = 0;   // input geometry (per example)
  int Ho = 0, Wo = 0, Co = 0; // output geometry
  int64_t w_off = -1, b_off = -1, nw = 0;
  bool stored = false;        // output activation kept in the workspace
  size_t act_off = 0;
  int64_t act_rs = 0;         // elements per replica of the output
  size_t gpre_off = 0, gin_off = 0, wf_off = 0, wd_off = 0;
  bool has_gin = false;
  int Kp = 0, Kdp = 0;
  int splits = 1, chunk = 0;
  bool no_relu = false;       // conv followed by a norm layer: raw output
  int groups = 0;             // group norm: groups (0: batch norm)
  int nstat = 0;              // norm statistics per replica
  int64_t st_off = 0;         // batch norm: running statistics in the state vector
  size_t mean_off = 0, rstd_off = 0, sums_off = 0;
  int blk = -1;               // GCPSL_BLOCK: its entry in Plan::blocks
  // conv followed by a stored 2 x 2 max pool and another conv: the forward
  // writes the pool's routing codes (one byte per pooled element) instead of
  // the unpooled output, and the layer's gradients take the next conv's
  // input gradient routed through them (no unpooled output or gradient)
  bool pcode = false;
  // the head conv (bf16, head of a max pool then the mean): its pooling
  // epilogue writes the max pool's routing codes and the head's pooling
  // backward routes through them, so its output is not kept (gpre is)
  bool hcode = false;
  size_t code_off = 0;
  // splits > 1: this layer's split-K partials of the weights and the biases,
  // in floats from Plan::off_part (the SGD pass sums them)
  size_t part_off = 0, dbpart_off = 0;
};

// A ResNet basic block (GCPSL_BLOCK) as internal layers, each with its own
// parameters, buffers and split-K plan in the LayerInfo fields the other
// layers use: c1 (3 x 3, the block's stride; at stride 2 on im2col rows of
// Kc1 = 9 cin columns) -> n1 (norm, ReLU) -> c2 (3 x 3) -> n2 (norm, + the
// shortcut, ReLU: its output and gradient are the block's); with a
// projection, cp (1 x 1, stride, on rows of the strided input) -> np (norm,
// no ReLU) is the shortcut.  At stride 2 the input gradients of c1 and cp
// take their output gradients spread back to the input grid (gup).
struct BlockInfo {
  int stride = 1;
  bool proj = false;
  int Kc1 = 0, Kcp = 0;
  LayerInfo c1, n1, c2, n2, cp, np;
  size_t cols1_off = 0, xs_off = 0, gup_off = 0, gsc_off = 0;
};

bool is_norm(int kind) { return kind == GCPSL_BATCHNORM || kind == GCPSL_GROUPNORM; }
// layers whose output is followed by ReLU and stored: conv, norm or block
bool is_act(int kind) { return kind == GCPSL_CONV3X3 || is_norm(kind) || kind == GCPSL_BLOCK; }

struct Plan {
  int dtype = 0, esz = 4;
  int K = 0, C = 0, B = 0, L = 0, H = 0, W = 0, Cin = 0;
  int64_t n_examples = 0, max_steps = 0;
  int max_window = 1;
  std::vector<LayerInfo> ly;
  std::vector<BlockInfo> blocks;
  int64_t P = 0, Pc = 0, S = 0;
  int head_conv = -1, avg_idx = -1, lin_idx = -1;  // head_conv: conv or norm feeding the head pooling
  bool head_maxpool = false;
  int Ch_head = 0;
  // The image layer's input is staged as im2col rows when its channel count
  // is not a whole number of 16-byte vectors: Kc columns per pixel.
  bool col0 = false;
  int Kc = 0;
  int64_t x_rs = 0;  // elements of one staged step: C * B * H * W * (Kc or Cin)
  int schedule = GCPSL_SCHED_LOCKSTEP;
  int cut = 0;
  size_t off_ids = 0, off_off = 0, off_coe = 0, off_fw = 0, off_hits = 0, off_idx = 0, off_y = 0,
         off_x = 0, off_dh = 0, off_grad = 0, off_part = 0, off_loss = 0, off_order = 0,
         off_ident = 0, off_npart = 0, off_dev = 0, off_ghist = 0, off_sgdseg = 0;
  // the SGD pass in segments of the parameter vector (SgdSeg): the split-K
  // partials of every split layer are summed there; uploaded at creation
  std::vector<SgdSeg> sgd_segs;
  int sgd_blocks = 0, sgd_vec = 1;
  double sgd_part_bytes = 0.0;  // partial floats the pass reads per step, in bytes
  size_t total = 0;
};

int build_plan(const gcpsl_desc *d, Plan &p) {
  if (!d) return gcpsl_fail(GCPSL_EINVAL, "null description");
  if (d->dtype != GCPSL_F32 && d->dtype != GCPSL_BF16) return gcpsl_fail(GCPSL_EINVAL, "unknown dtype");
  if (d->K < 1 || d->K > 65536) return gcpsl_fail(GCPSL_EINVAL, "K must be in [1, 65536]");
  if (d->C < 1 || d->C > 1024) return gcpsl_fail(GCPSL_EINVAL, "C must be in [1, 1024]");
  if (d->C > d->K) return gcpsl_fail(GCPSL_EINVAL, "C must not exceed K");
  if (d->B < 1 || d->L < 2 || d->H < 1 || d->W < 1 || d->Cin < 1)
    return gcpsl_fail(GCPSL_EINVAL, "B, L, H, W, Cin out of range");
  if (d->L > kMaxDevClasses) return gcpsl_fail(GCPSL_EUNSUPPORTED, "L must not exceed 4096");
  if (d->B >= (1 << 29)) return gcpsl_fail(GCPSL_EUNSUPPORTED, "B must be below 2^29");
  if (d->n_examples < 1 || d->n_examples > INT32_MAX)
    return gcpsl_fail(GCPSL_EINVAL, "n_examples must be in [1, 2^31)");
  if (d->max_steps < 1 || d->max_window < 1) return gcpsl_fail(GCPSL_EINVAL, "max_steps and max_window must be >= 1");
  if (d->schedule != GCPSL_SCHED_LOCKSTEP && d->schedule != GCPSL_SCHED_EPOCH)
    return gcpsl_fail(GCPSL_EINVAL, "unknown schedule");
  if (!d->layers || d->n_layers < 3) return gcpsl_fail(GCPSL_EINVAL, "need at least conv, avgpool, linear");
  {
    // weight-copy jobs (prep_add_layer): two per conv, at most
    int jobs = 0;
    for (int i = 0; i < d->n_layers; ++i) {
      jobs += d->layers[i].kind == GCPSL_CONV3X3 ? 2 : 0;
      if (d->layers[i].kind == GCPSL_BLOCK)
        jobs += 4 + ((d->layers[i].flags & GCPSL_STRIDE2) || d->layers[i].cin != d->layers[i].cout ? 2 : 0);
    }
    if (jobs > kMaxPrepJobs) return gcpsl_fail(GCPSL_EUNSUPPORTED, "too many conv layers (weight-copy jobs)");
  }
  if (d->cut < 1 || d->cut > d->n_layers - 2) return gcpsl_fail(GCPSL_EINVAL, "cut outside the model");
  if ((int64_t)d->B * d->H * d->W > INT32_MAX / 4) return gcpsl_fail(GCPSL_EUNSUPPORTED, "batch too large");

  p.dtype = d->dtype;
  p.esz = d->dtype == GCPSL_BF16 ? 2 : 4;
  p.K = d->K; p.C = d->C; p.B = d->B; p.L = d->L; p.H = d->H; p.W = d->W; p.Cin = d->Cin;
  p.n_examples = d->n_examples;
  p.schedule = d->schedule;
  p.max_steps = d->max_steps;
  p.max_window = d->max_window;
  p.cut = d->cut;
  const int n = d->n_layers;
  p.ly.assign(n, LayerInfo());
  int H = d->H, W = d->W, c = d->Cin;
  int64_t P = 0;
  for (int i = 0; i < n; ++i) {
    LayerInfo &l = p.ly[i];
    l.spec = d->layers[i];
    l.H = H; l.W = W; l.Ci = c;
    const int kind = l.spec.kind;
    if (kind == GCPSL_CONV3X3) {
      if (l.spec.cin != c) return gcpsl_fail(GCPSL_EINVAL, "conv cin does not match its input");
      if (!(c == 3 && i == 0) && c % 8 != 0)
        return gcpsl_fail(GCPSL_EUNSUPPORTED, "conv cin must be a multiple of 8 (or 3 for layer 0)");
      if (l.spec.cout < 8 || l.spec.cout % 8 != 0)
        return gcpsl_fail(GCPSL_EUNSUPPORTED, "conv cout must be a positive multiple of 8");
      if ((l.spec.flags & GCPSL_RESIDUAL) && l.spec.cin != l.spec.cout)
        return gcpsl_fail(GCPSL_EINVAL, "residual conv needs cin == cout");
      if (l.spec.flags & ~GCPSL_RESIDUAL) return gcpsl_fail(GCPSL_EINVAL, "unknown layer flag");
      if (i > 0 && !is_act(p.ly[i - 1].spec.kind) && p.ly[i - 1].spec.kind != GCPSL_MAXPOOL2)
        return gcpsl_fail(GCPSL_EUNSUPPORTED, "conv must follow a conv, a norm or a max pool");
      l.no_relu = i + 1 < n && is_norm(d->layers[i + 1].kind);
      if (l.no_relu && (l.spec.flags & GCPSL_RESIDUAL))
        return gcpsl_fail(GCPSL_EUNSUPPORTED, "a residual conv cannot feed a norm layer");
      l.Co = l.spec.cout; l.Ho = H; l.Wo = W;
      l.nw = (int64_t)l.Co * 9 * l.Ci;
      l.w_off = P; P += l.nw;
      l.b_off = P; P += l.Co;
      c = l.Co;
    } else if (is_norm(kind)) {
      if (i == 0 || p.ly[i - 1].spec.kind != GCPSL_CONV3X3)
        return gcpsl_fail(GCPSL_EUNSUPPORTED, "a norm layer must follow a conv");
      if (l.spec.cin != c || l.spec.cout != c) return gcpsl_fail(GCPSL_EINVAL, "norm channels must match the conv");
      l.groups = kind == GCPSL_GROUPNORM ? l.spec.groups : 0;
      if (kind == GCPSL_GROUPNORM && (l.groups < 1 || c % l.groups != 0))
        return gcpsl_fail(GCPSL_EINVAL, "group norm needs groups >= 1 dividing the channels");
      if (!norm_ok(d->dtype, c, l.groups)) return gcpsl_fail(GCPSL_EUNSUPPORTED, "norm layer channels");
      l.Co = c; l.Ho = H; l.Wo = W;
      l.w_off = P; P += c;  // gamma
      l.b_off = P; P += c;  // beta
      l.nstat = l.groups ? d->B * l.groups : c;
      if (kind == GCPSL_BATCHNORM) {
        l.st_off = p.S;
        p.S += 2 * c + 1;  // running mean, running variance, counter
      }
    } else if (kind == GCPSL_BLOCK) {
      const int cout = l.spec.cout;
      if (i == 0 || !is_act(p.ly[i - 1].spec.kind) || p.ly[i - 1].no_relu)
        return gcpsl_fail(GCPSL_EUNSUPPORTED, "a block must follow a conv, norm or block");
      if (l.spec.cin != c) return gcpsl_fail(GCPSL_EINVAL, "block cin does not match its input");
      if (c % 8 != 0 || cout < 8 || cout % 8 != 0)
        return gcpsl_fail(GCPSL_EUNSUPPORTED, "block channels must be multiples of 8");
      if (l.spec.flags & ~GCPSL_STRIDE2) return gcpsl_fail(GCPSL_EINVAL, "unknown block flag");
      const int st = (l.spec.flags & GCPSL_STRIDE2) ? 2 : 1;
      if (st == 2 && (H % 2 || W % 2)) return gcpsl_fail(GCPSL_EINVAL, "a stride-2 block needs even H and W");
      l.groups = l.spec.groups;
      if (l.groups < 0 || (l.groups && cout % l.groups) || !norm_ok(d->dtype, cout, l.groups))
        return gcpsl_fail(GCPSL_EUNSUPPORTED, "block norm channels / groups");
      BlockInfo bk;
      bk.stride = st;
      bk.proj = st != 1 || c != cout;
      l.blk = (int)p.blocks.size();
      l.Co = cout; l.Ho = H / st; l.Wo = W / st;
      // internal layers: input geometry, parameters (w, b, gamma, beta in the
      // order of the layer description), batch-norm state
      auto conv = [&](LayerInfo &cv, int ci, int co, int hh, int ww, int taps) {
        cv.spec = gcpsl_layer{GCPSL_CONV3X3, ci, co, 0, 0};
        cv.H = hh; cv.W = ww; cv.Ci = ci; cv.Co = co; cv.Ho = l.Ho; cv.Wo = l.Wo;
        cv.nw = (int64_t)co * taps * ci;
        cv.w_off = P; P += cv.nw;
        cv.b_off = P; P += co;
        cv.no_relu = true;
      };
      auto nrm = [&](LayerInfo &nl) {
        nl.spec = gcpsl_layer{l.groups ? GCPSL_GROUPNORM : GCPSL_BATCHNORM, cout, cout, 0, l.groups};
        nl.H = l.Ho; nl.W = l.Wo; nl.Ci = nl.Co = cout; nl.Ho = l.Ho; nl.Wo = l.Wo;
        nl.groups = l.groups;
        nl.w_off = P; P += cout;
        nl.b_off = P; P += cout;
        nl.nstat = l.groups ? d->B * l.groups : cout;
        if (!l.groups) {
          nl.st_off = p.S;
          p.S += 2 * cout + 1;
        }
      };
      conv(bk.c1, c, cout, H, W, 9);
      nrm(bk.n1);
      conv(bk.c2, cout, cout, l.Ho, l.Wo, 9);
      nrm(bk.n2);
      if (bk.proj) {
        conv(bk.cp, c, cout, H, W, 1);
        nrm(bk.np);
      }
      p.blocks.push_back(bk);
      H = l.Ho; W = l.Wo;
      c = cout;
    } else if (kind == GCPSL_MAXPOOL2) {
      if (i == 0 || !is_act(p.ly[i - 1].spec.kind))
        return gcpsl_fail(GCPSL_EUNSUPPORTED, "max pool must follow a conv or a norm layer");
      if (H % 2 || W % 2) return gcpsl_fail(GCPSL_EINVAL, "max pool needs even H and W");
      H /= 2; W /= 2;
      l.Co = c; l.Ho = H; l.Wo = W;
    } else if (kind == GCPSL_AVGPOOL) {
      if (i != n - 2) return gcpsl_fail(GCPSL_EUNSUPPORTED, "avgpool must be the second-to-last layer");
      l.Co = c; l.Ho = 1; l.Wo = 1;
    } else if (kind == GCPSL_LINEAR) {
      if (i != n - 1) return gcpsl_fail(GCPSL_EUNSUPPORTED, "linear must be the last layer");
      if (l.spec.cin != c || l.spec.cout != d->L)
        return gcpsl_fail(GCPSL_EINVAL, "linear must map the pooled channels to L classes");
      l.Co = l.spec.cout; l.Ho = 1; l.Wo = 1;
      l.nw = (int64_t)l.Co * l.Ci;
      l.w_off = P; P += l.nw;
      l.b_off = P; P += l.Co;
    } else {
      return gcpsl_fail(GCPSL_EINVAL, "unknown layer kind");
    }
    if (i == d->cut - 1) p.Pc = P;
  }
  if (d->layers[0].kind != GCPSL_CONV3X3) return gcpsl_fail(GCPSL_EUNSUPPORTED, "layer 0 must be a conv");
  p.P = P;
  p.avg_idx = n - 2;
  p.lin_idx = n - 1;
  if (p.ly[n - 3].spec.kind == GCPSL_MAXPOOL2) {
    p.head_maxpool = true;
    p.head_conv = n - 4;
  } else {
    p.head_conv = n - 3;
  }
  if (p.head_conv < 0 || !is_act(p.ly[p.head_conv].spec.kind) || p.ly[p.head_conv].no_relu)
    return gcpsl_fail(GCPSL_EUNSUPPORTED, "avgpool must follow a conv or norm layer, optionally + max pool");
  p.Ch_head = p.ly[p.head_conv].Co;
  if (!linear_ce_reg_ok(d->B, p.Ch_head, d->L) && linear_ce_lds_bytes(d->B, p.Ch_head, d->L) > kMaxLinearLds)
    return gcpsl_fail(GCPSL_EUNSUPPORTED, "classifier head too large for one workgroup (B * channels)");

  // workspace layout
  const int C = p.C, B = p.B;
  const int bk_tile = p.dtype == GCPSL_BF16 ? 64 : 32;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + bytes);
    return at;
  };
  p.off_ids = take(sizeof(int32_t) * p.n_examples);
  p.off_off = take(sizeof(int64_t) * (C + 1));
  p.off_coe = take(sizeof(int32_t) * p.n_examples);
  p.off_fw = take(sizeof(double) * C);
  p.off_order = take(sizeof(int32_t) * C);  // clusters by epoch rounds, descending
  p.off_ident = take(sizeof(int32_t) * C);  // 0, 1, ..., C-1
  p.off_hits = take(sizeof(int32_t) * p.max_steps * C);
  p.off_dev = take(sizeof(int64_t) * p.max_steps * C);  // batch deviation numerators (Sec. V-E)
  p.off_ghist = take(sizeof(int64_t) * p.L);           // examples per class in the data set
  p.off_idx = take(sizeof(int32_t) * (size_t)p.max_window * C * B);
  p.off_y = take(sizeof(int32_t) * (size_t)p.max_window * C * B);
  {
    // a first layer with few channels runs on im2col rows that the gather
    // writes (col0), unless its kernels build those rows from the gathered
    // images themselves (3 -> 32 channels, bf16, 32-pixel-wide images)
    const int vec = 16 / p.esz;
    const LayerInfo &l0 = p.ly[0];
    const bool img3 = !(l0.spec.flags & GCPSL_RESIDUAL) && conv_im3_ok(p.dtype, p.Cin, l0.Co, p.H, p.W);
    p.col0 = p.Cin % vec != 0 && !img3;
    p.Kc = p.col0 ? round_up(9 * p.Cin, vec) : p.Cin;
  }
  p.x_rs = (int64_t)C * B * p.H * p.W * p.Kc;
  p.off_x = take((size_t)p.esz * p.max_window * p.x_rs);
  size_t part = 0, npart = 0;
  std::vector<const LayerInfo *> split_layers;
  // split-K over pixels for a weight gradient of M pixels per replica with
  // Ci_eff columns per tap (taps 9, or 1 on im2col rows)
  auto plan_wgrad = [&](LayerInfo &l, int M, int Ci_eff, int taps, int Hh, int Ww) {
    int kt = wgrad_k_tile(p.dtype);
    int nkt = (M + kt - 1) / kt;
    int bm, bn;
    const int nwc = taps == 1 ? Ci_eff : 9 * Ci_eff;
    int splits;
    if (wgrad_lds_ok(p.dtype, l.Co, Ci_eff) || wgrad_col_ok(p.dtype, l.Co, Ci_eff, taps) ||
        (taps == 9 && conv_im3_ok(p.dtype, Ci_eff, l.Co, Hh, Ww))) {
      // Kernels that run one workgroup per CU (the halo weight gradients,
      // MFMA-bound): pick the split count that minimises the time in units
      // of one k tile of a workgroup on its CU, (workgroups / 256 CUs,
      // rounded up) x (k tiles per workgroup), plus writing and re-reading
      // all the partials (bm x bn floats per workgroup) at the chip's HBM
      // rate B: with F = 5.9 TFLOP/s reached per CU and B = 6 TB/s, the
      // 8 bytes of each partial float cost 4 F / (B kt) k tiles per partial
      // tile on the whole chip (the tile's size cancels).  The others (two
      // or four workgroups per CU, bound by their copies rather than the
      // MFMAs): (rounds of 256 x per_cu workgroups) x (k tiles per
      // workgroup + the cost of writing and re-reading a partial tile,
      // about 16 k tiles).
      int tile_bk, per_cu;
      wgrad_lds_tile(l.Co, Ci_eff, Hh, Ww, taps, &bm, &bn, &tile_bk, &per_cu);
      kt = tile_bk;  // chunks are whole k tiles of the kernel the layer runs
      nkt = (M + kt - 1) / kt;
      const int64_t tiles = (int64_t)((l.Co + bm - 1) / bm) * ((nwc + bn - 1) / bn) * C;
      const int64_t slots = 256 * (int64_t)per_cu;
      double best = -1.0;
      splits = 1;
      for (int sp = 1; sp <= std::min(64, nkt); ++sp) {
        const double ktiles = (double)((nkt + sp - 1) / sp);
        double cost;
        if (per_cu == 1)
          cost = (double)((tiles * sp + 255) / 256) * ktiles +
                 (sp > 1 ? (double)(tiles * sp) * 4.0 * 5.9e12 / (6.0e12 * kt) : 0.0);
        else
          cost = (double)((tiles * sp + slots - 1) / slots) * (ktiles + (sp > 1 ? 16.0 * 64 / kt : 0.0));
        if (best < 0 || cost < best) best = cost, splits = sp;
      }
    } else {
      wgrad_tile(p.dtype, l.Co, nwc, &bm, &bn);
      const int64_t tiles = (int64_t)((l.Co + bm - 1) / bm) * ((nwc + bn - 1) / bn) * C;
      const int64_t target = bm * bn >= 256 * 128 ? 512 : 1024;  // workgroups to fill 256 CUs
      splits = (int)std::min<int64_t>(std::max(1, nkt / 4), (target + tiles - 1) / tiles);
      splits = std::max(1, splits);
    }
    const int per = (nkt + splits - 1) / splits;
    l.chunk = per * kt;
    l.splits = (M + l.chunk - 1) / l.chunk;
    if (l.splits > 1) {  // its own partials, 16-byte aligned, weights then biases
      l.part_off = part;
      part = (part + (size_t)l.splits * C * l.nw + 3) / 4 * 4;
      l.dbpart_off = part;
      part = (part + (size_t)l.splits * C * l.Co + 3) / 4 * 4;
      split_layers.push_back(&l);
    }
  };
  // kernels address one replica's tensors with 32-bit byte offsets and mark
  // invalid lanes with offset 2^31
  auto small_enough = [&](int64_t px, int ci, int co, int taps) {
    return (int64_t)p.esz * px * std::max(ci, co) < (1ll << 31) &&
           (int64_t)p.esz * std::max(co, ci) * ((int64_t)taps * std::max(ci, co) + 64) < (1ll << 31);
  };
  // a norm layer's statistics buffers (output and gradient set by the caller)
  auto norm_buffers = [&](LayerInfo &l) {
    const int64_t rs = (int64_t)B * l.H * l.W;
    l.mean_off = take(sizeof(float) * C * l.nstat);
    l.rstd_off = take(sizeof(float) * C * l.nstat);
    l.sums_off = take(sizeof(double) * 2 * C * l.nstat);
    const int64_t chunks = (rs + norm_chunk(rs, C) - 1) / norm_chunk(rs, C);
    npart = std::max(npart, (size_t)(C * chunks * l.Co * 2));
  };
  // routing codes for conv i (LayerInfo::pcode): bf16, ReLU, a stored max
  // pool then a conv after it, and forward, input- and weight-gradient
  // kernels that take the codes for the layer's shape
  auto pool_codes = [&](int i) {
    const LayerInfo &l = p.ly[i];
    if (p.dtype != GCPSL_BF16 || l.spec.kind != GCPSL_CONV3X3 || l.no_relu || (l.spec.flags & GCPSL_RESIDUAL) ||
        i + 2 >= n || (i == 0 && p.col0))
      return false;
    if (p.ly[i + 1].spec.kind != GCPSL_MAXPOOL2 || (p.head_maxpool && i + 1 == n - 3) ||
        p.ly[i + 2].spec.kind != GCPSL_CONV3X3)
      return false;
    ConvArgs f{};
    f.epi = EPI_FWD;
    f.taps = 9;
    f.H = l.H; f.W = l.W; f.Csrc = l.Ci; f.N = l.Co; f.K = 9 * l.Ci; f.Kp = round_up(9 * l.Ci, bk_tile);
    if (!conv_fuses_pool(p.dtype, f) || !conv_pool_codes(p.dtype, f)) return false;
    if (i > 0) {
      ConvArgs g = f;
      g.epi = EPI_DGRAD;
      g.Csrc = l.Co; g.N = l.Ci; g.K = 9 * l.Co; g.Kp = round_up(9 * l.Co, bk_tile);
      if (!conv_pool_codes(p.dtype, g)) return false;
    }
    return wgrad_pool_codes(p.dtype, l.Co, l.Ci, l.H, l.W, 9);
  };
  // routing codes for the head conv (LayerInfo::hcode): bf16, the head's
  // mean of a 2 x 2 max pool written by the conv's own epilogue
  auto head_codes = [&](int i) {
    const LayerInfo &l = p.ly[i];
    if (p.dtype != GCPSL_BF16 || i != p.head_conv || !p.head_maxpool || l.spec.kind != GCPSL_CONV3X3 ||
        i + 2 != p.avg_idx)
      return false;
    ConvArgs f{};
    f.epi = EPI_FWD;
    f.taps = 9;
    f.H = l.H; f.W = l.W; f.Csrc = l.Ci; f.N = l.Co; f.K = 9 * l.Ci; f.Kp = round_up(9 * l.Ci, bk_tile);
    return conv_fuses_avg(p.dtype, f);
  };
  for (int i = 0; i < n; ++i) {
    LayerInfo &l = p.ly[i];
    const int kind = l.spec.kind;
    if (kind == GCPSL_BLOCK) {
      BlockInfo &bk = p.blocks[l.blk];
      const int64_t px_in = (int64_t)B * l.H * l.W, px = (int64_t)B * l.Ho * l.Wo;
      if (!small_enough(px_in, l.Ci, l.Co, 9) || !small_enough(px, 9 * l.Ci, l.Co, 1))
        return gcpsl_fail(GCPSL_EUNSUPPORTED, "per-replica layer tensors must stay below 2 GiB");
      auto out_buffers = [&](LayerInfo &x) {  // output and its gradient, [B][Ho][Wo][Co]
        x.stored = true;
        x.act_rs = px * x.Co;
        x.act_off = take((size_t)p.esz * C * x.act_rs);
        x.gpre_off = take((size_t)p.esz * C * x.act_rs);
      };
      auto weights = [&](LayerInfo &cv, int taps) {  // compute copies: forward rows, input-gradient rows
        cv.Kp = round_up(taps * cv.Ci, bk_tile);
        cv.wf_off = take((size_t)p.esz * C * cv.Co * cv.Kp);
        cv.Kdp = round_up(taps * cv.Co, bk_tile);
        cv.wd_off = take((size_t)p.esz * C * cv.Ci * cv.Kdp);
      };
      out_buffers(bk.c1);
      weights(bk.c1, 9);
      if (bk.stride == 2) {
        bk.Kc1 = 9 * l.Ci;
        bk.cols1_off = take((size_t)p.esz * C * px * bk.Kc1);
        plan_wgrad(bk.c1, (int)px, bk.Kc1, 1, l.Ho, l.Wo);
      } else {
        plan_wgrad(bk.c1, (int)px, l.Ci, 9, l.H, l.W);
      }
      out_buffers(bk.n1);
      norm_buffers(bk.n1);
      out_buffers(bk.c2);
      weights(bk.c2, 9);
      plan_wgrad(bk.c2, (int)px, l.Co, 9, l.Ho, l.Wo);
      // n2 writes the block's output; its gradient is the block's
      out_buffers(l);
      bk.n2.stored = true;
      bk.n2.act_rs = l.act_rs;
      bk.n2.act_off = l.act_off;
      bk.n2.gpre_off = l.gpre_off;
      norm_buffers(bk.n2);
      if (bk.proj) {
        bk.Kcp = l.Ci;
        bk.xs_off = take((size_t)p.esz * C * px * bk.Kcp);
        out_buffers(bk.cp);
        weights(bk.cp, 1);
        plan_wgrad(bk.cp, (int)px, bk.Kcp, 1, l.Ho, l.Wo);
        out_buffers(bk.np);  // (its gradient buffer is unused: np's gradient is the block's)
        norm_buffers(bk.np);
        bk.gsc_off = take((size_t)p.esz * C * px_in * l.Ci);
      }
      if (bk.stride == 2) bk.gup_off = take((size_t)p.esz * C * px_in * l.Co);
      continue;
    }
    if (is_norm(kind)) {
      const int64_t rs = (int64_t)B * l.H * l.W;
      l.stored = true;
      l.act_rs = rs * l.Co;
      l.act_off = take((size_t)p.esz * C * l.act_rs);
      l.gpre_off = take((size_t)p.esz * C * l.act_rs);  // dL/du
      norm_buffers(l);
      continue;
    }
    l.pcode = pool_codes(i);
    l.hcode = head_codes(i);
    if (l.pcode || l.hcode) {
      l.act_rs = (int64_t)B * l.Ho * l.Wo * l.Co;
      l.code_off = take((size_t)C * l.act_rs / 4);
    } else if (kind == GCPSL_CONV3X3 || (kind == GCPSL_MAXPOOL2 && !(p.head_maxpool && i == n - 3))) {
      l.stored = true;
      l.act_rs = (int64_t)B * l.Ho * l.Wo * l.Co;
      l.act_off = take((size_t)p.esz * C * l.act_rs);
    } else if (kind == GCPSL_AVGPOOL) {
      l.stored = true;
      l.act_rs = (int64_t)B * l.Co;
      l.act_off = take((size_t)p.esz * C * l.act_rs);
    }
    if (kind == GCPSL_CONV3X3) {
      const int64_t rs = (int64_t)B * l.H * l.W;
      if (!small_enough(rs, l.Ci, l.Co, 9))
        return gcpsl_fail(GCPSL_EUNSUPPORTED, "per-replica layer tensors must stay below 2 GiB");
      if (!l.pcode) l.gpre_off = take((size_t)p.esz * C * rs * l.Co);
      if (i > 0 && p.ly[i - 1].spec.kind == GCPSL_MAXPOOL2) {
        l.has_gin = true;
        l.gin_off = take((size_t)p.esz * C * rs * l.Ci);
      }
      l.Kp = round_up(9 * l.Ci, bk_tile);
      l.wf_off = take((size_t)p.esz * C * l.Co * l.Kp);
      if (i > 0) {
        l.Kdp = round_up(9 * l.Co, bk_tile);
        l.wd_off = take((size_t)p.esz * C * l.Ci * l.Kdp);
      }
      const bool col = i == 0 && p.col0;
      plan_wgrad(l, B * l.H * l.W, col ? p.Kc : l.Ci, col ? 1 : 9, l.H, l.W);
    }
  }
  p.off_dh = take(sizeof(float) * (size_t)C * B * p.Ch_head);
  p.off_grad = take(sizeof(float) * (size_t)C * p.P);
  p.off_part = take(sizeof(float) * std::max<size_t>(part, 1));
  {
    // SGD segments: each split layer's weights and biases from its partials,
    // the rest of the parameter vector from grad; kSgdBlockElems per block
    std::vector<SgdSeg> segs;
    for (const LayerInfo *l : split_layers) {
      segs.push_back(SgdSeg{l->w_off, l->nw, (int64_t)l->part_off, (int64_t)C * l->nw, l->nw, l->splits, 0});
      segs.push_back(SgdSeg{l->b_off, l->Co, (int64_t)l->dbpart_off, (int64_t)C * l->Co, l->Co, l->splits, 0});
      p.sgd_part_bytes += 4.0 * C * l->splits * (l->nw + l->Co);
    }
    std::sort(segs.begin(), segs.end(), [](const SgdSeg &a, const SgdSeg &b) { return a.begin < b.begin; });
    int64_t at = 0;
    for (const SgdSeg &g : segs) {
      if (g.begin < at) return gcpsl_fail(GCPSL_EUNSUPPORTED, "overlapping parameter segments");
      if (g.begin > at) p.sgd_segs.push_back(SgdSeg{at, g.begin - at, 0, 0, 0, 0, 0});
      p.sgd_segs.push_back(g);
      at = g.begin + g.len;
    }
    if (at > p.P) return gcpsl_fail(GCPSL_EUNSUPPORTED, "parameter segments beyond P");
    if (at < p.P) p.sgd_segs.push_back(SgdSeg{at, p.P - at, 0, 0, 0, 0, 0});
    p.sgd_vec = 4;
    for (const SgdSeg &g : p.sgd_segs) {
      const int64_t any = g.begin | g.len | g.src | g.ss | g.rs | p.P;
      while (any % p.sgd_vec) p.sgd_vec /= 2;
    }
    int64_t blocks = 0;
    for (SgdSeg &g : p.sgd_segs) {
      const int64_t be = g.splits > 0 ? 256 * p.sgd_vec : kSgdBlockElems;
      g.first_block = (int32_t)blocks;
      blocks += (g.len + be - 1) / be;
    }
    if (blocks > INT32_MAX / 2) return gcpsl_fail(GCPSL_EUNSUPPORTED, "parameter vector too long");
    p.sgd_blocks = (int)blocks;
    p.off_sgdseg = take(sizeof(SgdSeg) * p.sgd_segs.size());
  }
  p.off_loss = take(sizeof(float) * C);
  p.off_npart = take(sizeof(double) * std::max<size_t>(npart, 1));
  p.total = o;
  return GCPSL_OK;
}

}  // namespace

// Optional per-launch event timing (gcpsl_timing): every kernel launch is
// bracketed by two hipEvents on the caller's stream and tagged with the
// kernel instantiation and its algorithmic FLOPs and HBM bytes.
struct KernelRec {
  std::string name;
  double flops, bytes;
  size_t ev;
};

struct gcpsl_ctx {
  Plan plan;
  gcpsl_desc desc;
  std::vector<int64_t> sizes;
  std::vector<int64_t> rounds;  // r_n = floor(n_n / B)
  std::vector<int32_t> order;   // clusters by r_n descending, then index
  int64_t R = 0;                // max_n r_n: slots of a system epoch
  PrepJobs prep;                // weight-copy jobs of every conv layer
  char *ws = nullptr;
  int64_t staged_lo = -1;
  int staged_n = 0;
  int64_t horizon = 0;
  std::vector<int64_t> clients_in;  // |C_n|: clients of each cluster
  int static_dev = -1;              // device whose static workspace this context holds, or -1
  int64_t fusion_bytes = 0;         // logical payload of the fusions so far (Sec. V-E)
  bool timing = false;
  std::vector<hipEvent_t> events;
  size_t next_event = 0;
  std::vector<KernelRec> recs;
  template <typename T> T *at(size_t off) const { return reinterpret_cast<T *>(ws + off); }
  ~gcpsl_ctx() {
    for (hipEvent_t e : events) (void)hipEventDestroy(e);
  }
};

namespace {

// Start a timed launch: returns the event slot, or SIZE_MAX when timing is off.
size_t tbegin(gcpsl_ctx *ctx, hipStream_t s) {
  if (!ctx->timing) return SIZE_MAX;
  while (ctx->events.size() < ctx->next_event + 2) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return SIZE_MAX;
    ctx->events.push_back(e);
  }
  const size_t i = ctx->next_event;
  if (hipEventRecord(ctx->events[i], s) != hipSuccess) return SIZE_MAX;
  return i;
}

void tend(gcpsl_ctx *ctx, hipStream_t s, size_t i, const std::string &name, double flops, double bytes) {
  if (i == SIZE_MAX) return;
  if (hipEventRecord(ctx->events[i + 1], s) != hipSuccess) return;
  ctx->recs.push_back({name, flops, bytes, i});
  ctx->next_event = i + 2;
}

}  // namespace

// LAUNCH_T(name, flops, bytes, launch-expression): launch, time when enabled.
#define LAUNCH_T(NAME, FLOPS, BYTES, EXPR)                                                       \
  do {                                                                                          \
    const size_t t_ = tbegin(ctx, s);                                                           \
    const hipError_t e_ = (EXPR);                                                               \
    if (e_ != hipSuccess) return gcpsl_fail(GCPSL_EHIP, std::string("launch failed: ") + hipGetErrorString(e_)); \
    tend(ctx, s, t_, (NAME), (FLOPS), (BYTES));                                                 \
  } while (0)

extern "C" int gcpsl_param_count(const gcpsl_desc *d, int64_t *P, int64_t *P_client) {
  gcpsl_clear_error();
  Plan p;
  const int rc = build_plan(d, p);
  if (rc) return rc;
  if (P) *P = p.P;
  if (P_client) *P_client = p.Pc;
  return GCPSL_OK;
}

extern "C" int gcpsl_state_count(const gcpsl_desc *d, int64_t *S) {
  gcpsl_clear_error();
  if (!S) return gcpsl_fail(GCPSL_EINVAL, "null output");
  Plan p;
  const int rc = build_plan(d, p);
  if (rc) return rc;
  *S = p.S;
  return GCPSL_OK;
}

extern "C" int gcpsl_workspace_bytes(const gcpsl_desc *d, size_t *bytes) {
  gcpsl_clear_error();
  if (!bytes) return gcpsl_fail(GCPSL_EINVAL, "null output");
  Plan p;
  const int rc = build_plan(d, p);
  if (rc) return rc;
  *bytes = p.total;
  return GCPSL_OK;
}

#define HIP_TRY(expr)                                                                       \
  do {                                                                                      \
    const hipError_t e_ = (expr);                                                           \
    if (e_ != hipSuccess) return gcpsl_fail(GCPSL_EHIP, std::string(#expr ": ") + hipGetErrorString(e_)); \
  } while (0)

// The workspace of the allocation-free context (gcpsl_create_static): one
// array per device, held from the library's load until the process ends.  In
// host code `scratch` only names the symbol; its device address comes from
// hipGetSymbolAddress, once per device with that device current.
static __device__ __align__(256) char scratch[GCPSL_STATIC_WORKSPACE_BYTES];

namespace {
constexpr int kMaxStaticDevices = 64;
struct StaticWorkspaces {
  std::mutex mu;
  char *ptr[kMaxStaticDevices] = {};   // device address of `scratch` per device
  bool busy[kMaxStaticDevices] = {};   // a static context lives on the device
};
StaticWorkspaces g_static;

// Claims the current device's array for one context: its address, or an
// error (no device, lookup failed, already claimed).
int claim_static(int *dev_out, char **ptr_out) {
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxStaticDevices) return gcpsl_fail(GCPSL_EUNSUPPORTED, "device id beyond 63");
  std::lock_guard<std::mutex> lock(g_static.mu);
  if (g_static.busy[dev])
    return gcpsl_fail(GCPSL_ESTATE, "a static context already lives on device " + std::to_string(dev));
  if (!g_static.ptr[dev]) {
    void *a = nullptr;
    HIP_TRY(hipGetSymbolAddress(&a, HIP_SYMBOL(scratch)));
    if (!a || reinterpret_cast<uintptr_t>(a) % kAlign) return gcpsl_fail(GCPSL_EHIP, "static workspace address");
    g_static.ptr[dev] = reinterpret_cast<char *>(a);
  }
  g_static.busy[dev] = true;
  *dev_out = dev;
  *ptr_out = g_static.ptr[dev];
  return GCPSL_OK;
}

void release_static(int dev) {
  if (dev < 0 || dev >= kMaxStaticDevices) return;
  std::lock_guard<std::mutex> lock(g_static.mu);
  g_static.busy[dev] = false;
}

int create_ctx(const gcpsl_desc *d, char *ws, size_t ws_bytes, gcpsl_ctx **out);
}  // namespace

extern "C" int gcpsl_create(const gcpsl_desc *d, gcpsl_ctx **out) {
  gcpsl_clear_error();
  if (!out) return gcpsl_fail(GCPSL_EINVAL, "null output");
  *out = nullptr;
  if (!d) return gcpsl_fail(GCPSL_EINVAL, "null description");
  if (!d->workspace) return gcpsl_fail(GCPSL_EINVAL, "null pointer in description");
  return create_ctx(d, reinterpret_cast<char *>(d->workspace), d->workspace_bytes, out);
}

extern "C" int gcpsl_create_static(const gcpsl_desc *d, gcpsl_ctx **out) {
  gcpsl_clear_error();
  if (!out) return gcpsl_fail(GCPSL_EINVAL, "null output");
  *out = nullptr;
  Plan p;
  if (int rc = build_plan(d, p)) return rc;
  if (p.total > GCPSL_STATIC_WORKSPACE_BYTES)
    return gcpsl_fail(GCPSL_EINVAL, "the description needs " + std::to_string(p.total) +
                                        " workspace bytes, more than the static workspace's " +
                                        std::to_string((size_t)GCPSL_STATIC_WORKSPACE_BYTES));
  int dev = -1;
  char *ws = nullptr;
  if (int rc = claim_static(&dev, &ws)) return rc;
  const int rc = create_ctx(d, ws, GCPSL_STATIC_WORKSPACE_BYTES, out);
  if (rc) {
    release_static(dev);
    return rc;
  }
  (*out)->static_dev = dev;
  return GCPSL_OK;
}

namespace {
int create_ctx(const gcpsl_desc *d, char *ws, size_t ws_bytes, gcpsl_ctx **out) {
  Plan p;
  int rc = build_plan(d, p);
  if (rc) return rc;
  if (!d->client_of_example || !d->cluster_of_client || !d->images || !d->labels || !d->theta ||
      !d->momentum_buf)
    return gcpsl_fail(GCPSL_EINVAL, "null pointer in description");
  if (reinterpret_cast<uintptr_t>(ws) % kAlign)
    return gcpsl_fail(GCPSL_EINVAL, "workspace must be 256-byte aligned");
  if (reinterpret_cast<uintptr_t>(d->theta) % 16 || reinterpret_cast<uintptr_t>(d->momentum_buf) % 16)
    return gcpsl_fail(GCPSL_EINVAL, "theta and momentum must be 16-byte aligned");
  if (p.S > 0 && !d->norm_state) return gcpsl_fail(GCPSL_EINVAL, "the model has batch norm layers: norm_state needed");
  if (ws_bytes < p.total)
    return gcpsl_fail(GCPSL_EINVAL, "workspace too small: need " + std::to_string(p.total) + " bytes");
  if (!std::isfinite(d->lr) || !std::isfinite(d->momentum)) return gcpsl_fail(GCPSL_EINVAL, "lr and momentum must be finite");
  if (!(d->weight_decay >= 0.f) || !std::isfinite(d->weight_decay))
    return gcpsl_fail(GCPSL_EINVAL, "weight_decay must be finite and >= 0");
  if (d->nesterov != 0 && d->nesterov != 1) return gcpsl_fail(GCPSL_EINVAL, "nesterov must be 0 or 1");
  if (!(d->label_smoothing >= 0.f && d->label_smoothing < 1.f))
    return gcpsl_fail(GCPSL_EINVAL, "label_smoothing must lie in [0, 1)");
  for (int32_t k = 0; k < d->K; ++k)
    if (d->cluster_of_client[k] < 0 || d->cluster_of_client[k] >= d->C)
      return gcpsl_fail(GCPSL_EINVAL, "cluster_of_client out of range");
  // per-cluster example lists in ascending global id (CSR)
  std::vector<int64_t> off(p.C + 1, 0);
  for (int64_t e = 0; e < d->n_examples; ++e) {
    const int32_t k = d->client_of_example[e];
    if (k < 0 || k >= d->K) return gcpsl_fail(GCPSL_EINVAL, "client_of_example out of range");
    off[d->cluster_of_client[k] + 1] += 1;
  }
  for (int n = 0; n < p.C; ++n) {
    if (off[n + 1] < p.B)
      return gcpsl_fail(GCPSL_EINVAL, "cluster " + std::to_string(n) + " holds " +
                                          std::to_string(off[n + 1]) + " < B examples");
    off[n + 1] += off[n];
  }
  std::vector<int32_t> ids(d->n_examples);
  std::vector<int64_t> fill(off.begin(), off.end() - 1);
  for (int64_t e = 0; e < d->n_examples; ++e) ids[fill[d->cluster_of_client[d->client_of_example[e]]]++] = (int32_t)e;
  std::vector<double> fw(p.C);
  std::vector<int64_t> sizes(p.C);
  for (int n = 0; n < p.C; ++n) {
    sizes[n] = off[n + 1] - off[n];
    fw[n] = (double)sizes[n];
  }
  // class histogram of the data set (batch deviation, Sec. V-E); the labels
  // are checked here because the sampler counts them in LDS
  std::vector<int32_t> lab(d->n_examples);
  HIP_TRY(hipMemcpy(lab.data(), d->labels, sizeof(int32_t) * lab.size(), hipMemcpyDeviceToHost));
  std::vector<int64_t> ghist(p.L, 0);
  for (int64_t e = 0; e < d->n_examples; ++e) {
    if (lab[e] < 0 || lab[e] >= p.L) return gcpsl_fail(GCPSL_EINVAL, "labels must lie in [0, L)");
    ghist[lab[e]] += 1;
  }
  std::vector<int64_t> clients_in(p.C, 0);
  for (int32_t k = 0; k < d->K; ++k) clients_in[d->cluster_of_client[k]] += 1;
  HIP_TRY(hipMemcpy(ws + p.off_ghist, ghist.data(), sizeof(int64_t) * ghist.size(), hipMemcpyHostToDevice));
  HIP_TRY(hipMemset(ws + p.off_dev, 0xff, sizeof(int64_t) * p.max_steps * p.C));  // -1: no batch recorded
  HIP_TRY(hipMemcpy(ws + p.off_ids, ids.data(), sizeof(int32_t) * ids.size(), hipMemcpyHostToDevice));
  HIP_TRY(hipMemcpy(ws + p.off_off, off.data(), sizeof(int64_t) * off.size(), hipMemcpyHostToDevice));
  HIP_TRY(hipMemcpy(ws + p.off_coe, d->client_of_example, sizeof(int32_t) * d->n_examples, hipMemcpyHostToDevice));
  HIP_TRY(hipMemcpy(ws + p.off_fw, fw.data(), sizeof(double) * fw.size(), hipMemcpyHostToDevice));
  HIP_TRY(hipMemset(ws + p.off_hits, 0, sizeof(int32_t) * p.max_steps * p.C));
  // epoch schedule: the clusters taking a round at slot t are those with
  // r_n > t, a prefix of `order`
  std::vector<int64_t> rounds(p.C);
  std::vector<int32_t> order(p.C), ident(p.C);
  for (int n = 0; n < p.C; ++n) {
    rounds[n] = sizes[n] / p.B;
    order[n] = ident[n] = n;
  }
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return rounds[a] > rounds[b]; });
  HIP_TRY(hipMemcpy(ws + p.off_order, order.data(), sizeof(int32_t) * p.C, hipMemcpyHostToDevice));
  HIP_TRY(hipMemcpy(ws + p.off_ident, ident.data(), sizeof(int32_t) * p.C, hipMemcpyHostToDevice));
  HIP_TRY(hipMemcpy(ws + p.off_sgdseg, p.sgd_segs.data(), sizeof(SgdSeg) * p.sgd_segs.size(), hipMemcpyHostToDevice));
  gcpsl_ctx *ctx = new gcpsl_ctx();
  ctx->plan = std::move(p);
  ctx->desc = *d;
  ctx->desc.layers = nullptr;
  ctx->desc.client_of_example = nullptr;
  ctx->desc.cluster_of_client = nullptr;
  ctx->sizes = std::move(sizes);
  ctx->clients_in = std::move(clients_in);
  ctx->R = rounds[order[0]];
  ctx->rounds = std::move(rounds);
  ctx->order = std::move(order);
  ctx->ws = ws;
  for (size_t i = 0; i < ctx->plan.ly.size(); ++i) {
    const LayerInfo &l = ctx->plan.ly[i];
    if (l.spec.kind == GCPSL_CONV3X3)
      prep_add_layer(ctx->prep, l.w_off, l.Co, l.Ci, ws + l.wf_off, l.Kp, i > 0 ? ws + l.wd_off : nullptr, l.Kdp);
    if (l.spec.kind == GCPSL_BLOCK) {
      const BlockInfo &bk = ctx->plan.blocks[l.blk];
      for (const LayerInfo *cv : {&bk.c1, &bk.c2})
        prep_add_layer(ctx->prep, cv->w_off, cv->Co, cv->Ci, ws + cv->wf_off, cv->Kp, ws + cv->wd_off, cv->Kdp);
      if (bk.proj)
        prep_add_layer(ctx->prep, bk.cp.w_off, bk.cp.Co, bk.cp.Ci, ws + bk.cp.wf_off, bk.cp.Kp, ws + bk.cp.wd_off,
                       bk.cp.Kdp, 1);
    }
  }
  *out = ctx;
  return GCPSL_OK;
}
}  // namespace

extern "C" void gcpsl_destroy(gcpsl_ctx *ctx) {
  if (!ctx) return;
  release_static(ctx->static_dev);
  delete ctx;
}

extern "C" int gcpsl_cluster_sizes(gcpsl_ctx *ctx, int64_t *sizes) {
  gcpsl_clear_error();
  if (!ctx || !sizes) return gcpsl_fail(GCPSL_EINVAL, "null argument");
  std::copy(ctx->sizes.begin(), ctx->sizes.end(), sizes);
  return GCPSL_OK;
}

#define LAUNCH(expr)                                                                      \
  do {                                                                                    \
    const hipError_t e_ = (expr);                                                         \
    if (e_ != hipSuccess) return gcpsl_fail(GCPSL_EHIP, std::string("launch failed: ") + hipGetErrorString(e_)); \
  } while (0)

extern "C" int gcpsl_sample(gcpsl_ctx *ctx, int64_t step, int32_t nsteps, int32_t *idx_out, void *stream) {
  gcpsl_clear_error();
  if (!ctx) return gcpsl_fail(GCPSL_EINVAL, "null context");
  const Plan &p = ctx->plan;
  if (step < 0) return gcpsl_fail(GCPSL_EINVAL, "step must be >= 0");
  if (nsteps < 1 || nsteps > p.max_window) return gcpsl_fail(GCPSL_EINVAL, "nsteps outside [1, max_window]");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  int32_t *idx = ctx->at<int32_t>(p.off_idx);
  const double rows = (double)nsteps * p.C * p.B, row_elems = (double)p.H * p.W * p.Cin;
  LAUNCH_T("sample", 0.0, rows * 20.0,
           launch_sample(ctx->at<int32_t>(p.off_ids), ctx->at<int64_t>(p.off_off), ctx->at<int32_t>(p.off_coe),
                         ctx->desc.labels, ctx->at<int64_t>(p.off_ghist), idx, ctx->at<int32_t>(p.off_y),
                         ctx->at<int32_t>(p.off_hits), ctx->at<int64_t>(p.off_dev), p.C, p.B, p.K, p.L,
                         p.n_examples, ctx->desc.seed, step, nsteps, p.max_steps,
                         p.schedule == GCPSL_SCHED_EPOCH ? ctx->R : 0, s));
  if (p.col0)
    LAUNCH_T(p.dtype == GCPSL_BF16 ? "gather_im2col<bf16>" : "gather_im2col<f32>", 0.0,
             rows * (4.0 + row_elems * 4 + (double)p.H * p.W * p.Kc * p.esz),
             launch_gather_im2col(ctx->desc.images, idx, ctx->ws + p.off_x, p.dtype, (int64_t)nsteps * p.C * p.B,
                                  p.H, p.W, p.Cin, p.Kc, s));
  else
    LAUNCH_T(p.dtype == GCPSL_BF16 ? "gather<bf16>" : "gather<f32>", 0.0, rows * (4.0 + row_elems * (4 + p.esz)),
             launch_gather(ctx->desc.images, idx, ctx->ws + p.off_x, p.dtype, (int64_t)nsteps * p.C * p.B,
                           (int64_t)p.H * p.W * p.Cin, s));
  if (idx_out)
    HIP_TRY(hipMemcpyAsync(idx_out, idx, sizeof(int32_t) * (size_t)nsteps * p.C * p.B, hipMemcpyDeviceToDevice, s));
  ctx->staged_lo = step;
  ctx->staged_n = nsteps;
  return GCPSL_OK;
}

namespace {

// One local round of the replicas listed in rmap (device, nrep entries; null
// = replicas 0..nrep-1): every launch runs nrep replica slots.  The split-K
// plan of each layer is fixed at create, so a replica's arithmetic does not
// depend on which other replicas share the launches.
int run_round(gcpsl_ctx *ctx, int64_t step, const int32_t *rmap, int nrep, float *loss_out, hipStream_t s) {
  const Plan &p = ctx->plan;
  const gcpsl_desc &d = ctx->desc;
  const int C = nrep, B = p.B, n = (int)p.ly.size();
  const int64_t slot = step - ctx->staged_lo;
  char *ws = ctx->ws;
  const void *x_in = ws + p.off_x + (size_t)p.esz * slot * p.x_rs;
  const int32_t *y = ctx->at<int32_t>(p.off_y) + slot * p.C * B;
  float *grad = ctx->at<float>(p.off_grad);
  float *loss = loss_out ? loss_out : ctx->at<float>(p.off_loss);

  // compute copies of the conv weights (one launch for every layer)
  {
    double pb = 0.0;
    for (int i = 0; i < n; ++i) {
      const LayerInfo &l = p.ly[i];
      if (l.spec.kind == GCPSL_BLOCK) {
        const BlockInfo &bk = p.blocks[l.blk];
        for (const LayerInfo *cv : {&bk.c1, &bk.c2, &bk.cp})
          if (cv->nw) pb += (double)C * (8.0 * cv->nw + p.esz * ((double)cv->Co * cv->Kp + (double)cv->Ci * cv->Kdp));
      }
      if (l.spec.kind != GCPSL_CONV3X3) continue;
      pb += (double)C * ((i > 0 ? 8.0 : 4.0) * l.nw + p.esz * ((double)l.Co * l.Kp + (i > 0 ? (double)l.Ci * l.Kdp : 0.0)));
    }
    LAUNCH_T("prep_weights", 0.0, pb, launch_prep_weights(p.dtype, d.theta, p.P, C, rmap, ctx->prep, s));
  }

  // forward: client segment to the cut, server segment to the loss
  auto input_of = [&](int i) -> const void * { return i == 0 ? x_in : (const void *)(ws + p.ly[i - 1].act_off); };
  auto norm_args = [&](int i) {
    const LayerInfo &l = p.ly[i];
    const LayerInfo &cv = p.ly[i - 1];
    NormArgs na{};
    na.z = ws + cv.act_off;
    na.a = ws + l.act_off;
    na.du = ws + l.gpre_off;
    na.dz = ws + cv.gpre_off;
    na.mean = ctx->at<float>(l.mean_off);
    na.rstd = ctx->at<float>(l.rstd_off);
    na.part = ctx->at<double>(p.off_npart);
    na.sums = ctx->at<double>(l.sums_off);
    na.theta = d.theta;
    na.grad = grad;
    na.state = d.norm_state;
    na.P = p.P; na.g_off = l.w_off; na.b_off = l.b_off; na.S = p.S; na.st_off = l.st_off; na.z_rs = l.act_rs;
    na.Bt = B; na.H = l.H; na.W = l.W; na.Ch = l.Co; na.groups = l.groups; na.nstat = l.nstat;
    na.chunk_px = norm_chunk((int64_t)B * l.H * l.W, C);
    na.chunks = (int)(((int64_t)B * l.H * l.W + na.chunk_px - 1) / na.chunk_px);
    na.C = C;
    na.rmap = rmap;
    return na;
  };
  // ---- the pieces a block (GCPSL_BLOCK) runs, on its internal layers
  auto nargs = [&](const LayerInfo &nl, const void *z, void *out, const void *du, void *dz, const void *res,
                   int relu) {
    NormArgs na{};
    na.z = z;
    na.a = out;
    na.du = du;
    na.dz = dz;
    na.mean = ctx->at<float>(nl.mean_off);
    na.rstd = ctx->at<float>(nl.rstd_off);
    na.part = ctx->at<double>(p.off_npart);
    na.sums = ctx->at<double>(nl.sums_off);
    na.theta = d.theta;
    na.grad = grad;
    na.state = d.norm_state;
    na.P = p.P; na.g_off = nl.w_off; na.b_off = nl.b_off; na.S = p.S; na.st_off = nl.st_off;
    na.z_rs = (int64_t)B * nl.H * nl.W * nl.Co;
    na.Bt = B; na.H = nl.H; na.W = nl.W; na.Ch = nl.Co; na.groups = nl.groups; na.nstat = nl.nstat;
    na.chunk_px = norm_chunk((int64_t)B * nl.H * nl.W, C);
    na.chunks = (int)(((int64_t)B * nl.H * nl.W + na.chunk_px - 1) / na.chunk_px);
    na.C = C;
    na.rmap = rmap;
    na.res = res;
    na.relu = relu;
    return na;
  };
  // forward of an internal conv (raw output: a norm follows) over Hh x Ww
  // pixels: 3 x 3 stride 1 (taps 9) or a one-tap product on im2col rows
  auto conv_fwd = [&](const LayerInfo &cv, const void *src, int taps, int Csrc, int Hh, int Ww, void *out) -> int {
    ConvArgs a{};
    a.src = src;
    a.wt = ws + cv.wf_off;
    a.out = out;
    a.bias = d.theta + cv.b_off;
    a.Bt = B; a.H = Hh; a.W = Ww; a.N = cv.Co; a.Kp = cv.Kp;
    a.Csrc = Csrc;
    a.K = taps == 1 ? Csrc : 9 * Csrc;
    a.taps = taps;
    a.src_rs = (int64_t)B * Hh * Ww * Csrc;
    a.wt_rs = (int64_t)cv.Co * cv.Kp;
    a.out_rs = (int64_t)B * Hh * Ww * cv.Co;
    a.bias_rs = p.P;
    a.C = C;
    a.rmap = rmap;
    a.epi = EPI_FWD;
    a.no_relu = 1;
    std::string lab;
    const double M = (double)B * Hh * Ww;
    const double kk = (double)cv.nw / cv.Co;  // taps x input channels of the layer
    size_t t_ = tbegin(ctx, s);
    LAUNCH(launch_conv(p.dtype, a, s, &lab));
    tend(ctx, s, t_, lab, 2.0 * C * M * cv.Co * kk,
         (double)C * (p.esz * (M * Csrc + cv.Co * kk + M * cv.Co) + 4.0 * cv.Co));
    return GCPSL_OK;
  };
  // input gradient of an internal conv over the input grid Hh x Ww: out =
  // (sum + res) * [mask > 0] (res, mask optional); taps 9 (3 x 3 stride 1)
  // or 1 (1 x 1)
  auto conv_dgrad = [&](const LayerInfo &cv, const void *src, int taps, int Hh, int Ww, void *out, const void *res,
                        const void *mask) -> int {
    ConvArgs a{};
    a.src = src;
    a.wt = ws + cv.wd_off;
    a.out = out;
    a.res = res;
    a.mask = mask;
    a.Bt = B; a.H = Hh; a.W = Ww; a.Csrc = cv.Co; a.N = cv.Ci; a.K = taps * cv.Co; a.Kp = cv.Kdp;
    a.src_rs = (int64_t)B * Hh * Ww * cv.Co;
    a.wt_rs = (int64_t)cv.Ci * cv.Kdp;
    a.out_rs = (int64_t)B * Hh * Ww * cv.Ci;
    a.C = C;
    a.rmap = rmap;
    a.epi = EPI_DGRAD;
    a.taps = taps;
    std::string lab;
    const double M = (double)B * Hh * Ww;
    size_t t_ = tbegin(ctx, s);
    LAUNCH(launch_conv(p.dtype, a, s, &lab));
    tend(ctx, s, t_, lab, 2.0 * C * M * cv.Ci * taps * cv.Co,
         (double)C * p.esz * (M * cv.Co + (double)cv.Ci * taps * cv.Co + M * cv.Ci * (1 + (res ? 1 : 0) + (mask ? 1 : 0))));
    return GCPSL_OK;
  };
  // weight and bias gradient of a conv from g (Hh x Ww pixels) and its input
  // x (taps 9: the layer input, Ci_eff its channels; taps 1: im2col rows of
  // Ci_eff columns), split over pixels as planned, partials summed in order
  auto wgrad_run = [&](const LayerInfo &cv, const void *g, const void *x, int taps, int Ci_eff, int Hh,
                       int Ww) -> int {
    WgradArgs w{};
    w.g = g;
    w.x = x;
    w.Bt = B; w.H = Hh; w.W = Ww; w.Co = cv.Co;
    w.Ci = Ci_eff;
    w.taps = taps;
    w.nw = (int)(cv.nw / cv.Co);
    w.g_rs = (int64_t)B * Hh * Ww * cv.Co;
    w.x_rs = (int64_t)B * Hh * Ww * Ci_eff;
    w.C = C;
    w.rmap = rmap;
    w.splits = cv.splits;
    w.chunk = cv.chunk;
    if (cv.splits == 1) {
      w.dw = grad + cv.w_off; w.dw_rs = p.P; w.dw_ss = 0;
      w.db = grad + cv.b_off; w.db_rs = p.P; w.db_ss = 0;
    } else {  // the layer's own partials, summed by the SGD pass
      w.dw = ctx->at<float>(p.off_part) + cv.part_off; w.dw_rs = cv.nw; w.dw_ss = (int64_t)p.C * cv.nw;
      w.db = ctx->at<float>(p.off_part) + cv.dbpart_off; w.db_rs = cv.Co; w.db_ss = (int64_t)p.C * cv.Co;
    }
    {
      std::string lab;
      const double M = (double)B * Hh * Ww;
      size_t t_ = tbegin(ctx, s);
      LAUNCH(launch_wgrad(p.dtype, w, s, &lab));
      tend(ctx, s, t_, lab, 2.0 * C * M * cv.nw,
           (double)C * (p.esz * M * (cv.Co + cv.Ci) + 4.0 * cv.splits * (cv.nw + cv.Co)));
    }
    return GCPSL_OK;
  };
  bool pool_done = false;  // the max pool after the last conv was written by it
  bool avg_done = false;   // the head's mean pooling was written by the conv before it
  for (int i = 0; i < n; ++i) {
    const LayerInfo &l = p.ly[i];
    const int kind = l.spec.kind;
    if (kind == GCPSL_CONV3X3) {
      ConvArgs a{};
      a.src = input_of(i);
      a.wt = ws + l.wf_off;
      a.out = ws + l.act_off;
      a.bias = d.theta + l.b_off;
      a.res = (l.spec.flags & GCPSL_RESIDUAL) ? a.src : nullptr;
      a.mask = nullptr;
      const bool col = i == 0 && p.col0;
      a.Bt = B; a.H = l.H; a.W = l.W; a.N = l.Co; a.Kp = l.Kp;
      a.Csrc = col ? p.Kc : l.Ci;
      a.K = col ? p.Kc : 9 * l.Ci;
      a.taps = col ? 1 : 9;
      a.src_rs = (int64_t)B * l.H * l.W * a.Csrc;
      a.wt_rs = (int64_t)l.Co * l.Kp;
      a.out_rs = l.act_rs;
      a.bias_rs = p.P;
      a.C = C;
      a.rmap = rmap;
      a.epi = EPI_FWD;
      a.no_relu = l.no_relu ? 1 : 0;
      // a stored 2 x 2 max pool right after this conv: written by the conv
      // kernel itself where it supports that
      pool_done = false;
      if (i + 1 < n && p.ly[i + 1].spec.kind == GCPSL_MAXPOOL2 && p.ly[i + 1].stored && !l.no_relu) {
        a.pool_out = ws + p.ly[i + 1].act_off;
        a.pool_rs = p.ly[i + 1].act_rs;
        pool_done = conv_fuses_pool(p.dtype, a);
        if (!pool_done) a.pool_out = nullptr;
        if (l.pcode) {  // the pool and its routing codes only
          if (!pool_done) return gcpsl_fail(GCPSL_EUNSUPPORTED, "routing codes without the fused pool");
          a.pool_code = reinterpret_cast<uint8_t *>(ws + l.code_off);
          a.out = nullptr;
        }
      }
      // the head's mean pooling right after this conv: written by the conv
      // kernel itself where it supports that
      avg_done = false;
      if (i == p.head_conv && i + (p.head_maxpool ? 2 : 1) == p.avg_idx) {
        a.pool_out = ws + p.ly[p.avg_idx].act_off;
        a.pool_rs = (int64_t)B * l.Co;
        a.pool_max = p.head_maxpool ? 1 : 0;
        avg_done = conv_fuses_avg(p.dtype, a);
        if (!avg_done) a.pool_out = nullptr;
        if (l.hcode) {  // the mean and the max pool's routing codes only
          if (!avg_done) return gcpsl_fail(GCPSL_EUNSUPPORTED, "head routing codes without the fused pooling");
          a.pool_code = reinterpret_cast<uint8_t *>(ws + l.code_off);
          a.code_rs = l.act_rs / 4;
          a.out = nullptr;
        }
      }
      std::string lab;
      const double M = (double)B * l.H * l.W;
      const double fl = 2.0 * C * M * l.Co * 9.0 * l.Ci;
      const bool codes = l.pcode || l.hcode;
      const double by = (double)C * (p.esz * (M * l.Ci + (double)l.Co * 9 * l.Ci +
                                                (codes ? 0.0 : M * l.Co) + (a.res ? M * l.Co : 0.0) +
                                                (pool_done ? M / 4 * l.Co : 0.0) + (avg_done ? (double)B * l.Co : 0.0)) +
                                     (codes ? M / 4 * l.Co : 0.0) + 4.0 * l.Co);
      size_t t_ = tbegin(ctx, s);
      LAUNCH(launch_conv(p.dtype, a, s, &lab));
      tend(ctx, s, t_, lab, fl, by);
    } else if (kind == GCPSL_BLOCK) {
      // conv1 (the block's stride) -> norm1 + ReLU -> conv2 -> norm2 + shortcut + ReLU
      const BlockInfo &bk = p.blocks[l.blk];
      const void *x = input_of(i);
      const char *nn = l.groups ? "groupnorm_fwd" : "batchnorm_fwd";
      pool_done = avg_done = false;  // a max pool or the head after a block: their own kernels
      const double nby = (double)C * p.esz * B * l.Ho * l.Wo * l.Co * 3.0;
      if (bk.stride == 2) {
        LAUNCH_T("im2col", 0.0, (double)C * p.esz * B * l.Ho * l.Wo * (bk.Kc1 + 9.0 * l.Ci),
                 launch_im2col(p.dtype, x, ws + bk.cols1_off, C, rmap, B, l.H, l.W, l.Ci, l.Ho, l.Wo, 3, 3, 2, 1,
                               bk.Kc1, s));
        if (int rc = conv_fwd(bk.c1, ws + bk.cols1_off, 1, bk.Kc1, l.Ho, l.Wo, ws + bk.c1.act_off)) return rc;
      } else {
        if (int rc = conv_fwd(bk.c1, x, 9, l.Ci, l.H, l.W, ws + bk.c1.act_off)) return rc;
      }
      LAUNCH_T(nn, 0.0, nby, launch_norm_fwd(p.dtype, nargs(bk.n1, ws + bk.c1.act_off, ws + bk.n1.act_off, nullptr,
                                                             nullptr, nullptr, 1), s));
      if (int rc = conv_fwd(bk.c2, ws + bk.n1.act_off, 9, l.Co, l.Ho, l.Wo, ws + bk.c2.act_off)) return rc;
      const void *sc = x;
      if (bk.proj) {
        LAUNCH_T("im2col", 0.0, (double)C * p.esz * B * l.Ho * l.Wo * 2.0 * bk.Kcp,
                 launch_im2col(p.dtype, x, ws + bk.xs_off, C, rmap, B, l.H, l.W, l.Ci, l.Ho, l.Wo, 1, 1, bk.stride, 0,
                               bk.Kcp, s));
        if (int rc = conv_fwd(bk.cp, ws + bk.xs_off, 1, bk.Kcp, l.Ho, l.Wo, ws + bk.cp.act_off)) return rc;
        LAUNCH_T(nn, 0.0, nby, launch_norm_fwd(p.dtype, nargs(bk.np, ws + bk.cp.act_off, ws + bk.np.act_off, nullptr,
                                                               nullptr, nullptr, 0), s));
        sc = ws + bk.np.act_off;
      }
      LAUNCH_T(nn, 0.0, nby * 4.0 / 3.0, launch_norm_fwd(p.dtype, nargs(bk.n2, ws + bk.c2.act_off, ws + l.act_off,
                                                                         nullptr, nullptr, sc, 1), s));
    } else if (is_norm(kind)) {
      const double by = (double)C * p.esz * B * l.H * l.W * l.Co * (l.groups ? 3.0 : 3.0);
      LAUNCH_T(l.groups ? "groupnorm_fwd" : "batchnorm_fwd", 0.0, by, launch_norm_fwd(p.dtype, norm_args(i), s));
    } else if (kind == GCPSL_MAXPOOL2) {
      if (!l.stored) continue;  // fused into the head
      if (pool_done) continue;  // written by the conv before it
      LAUNCH_T("maxpool_fwd", 0.0, 1.25 * p.esz * (double)C * B * l.H * l.W * l.Ci,
               launch_maxpool_fwd(p.dtype, input_of(i), ws + l.act_off, C, rmap, B, l.H, l.W, l.Ci, s));
    } else if (kind == GCPSL_AVGPOOL) {
      if (avg_done) continue;  // written by the conv before it
      const LayerInfo &hc = p.ly[p.head_conv];
      LAUNCH_T("head_pool", 0.0, (double)p.esz * C * B * hc.Co * ((double)hc.Ho * hc.Wo + 1),
               launch_head_pool(p.dtype, ws + hc.act_off, ws + l.act_off, C, rmap, B, hc.Ho, hc.Wo, hc.Co,
                                p.head_maxpool ? 1 : 0, s));
    } else if (kind == GCPSL_LINEAR) {
      LAUNCH_T("linear_ce", 6.0 * C * B * l.Ci * l.Co,
               (double)C * (p.esz * B * l.Ci + 4.0 * (2.0 * l.nw + B * l.Ci + B)),
               launch_linear_ce(p.dtype, ws + p.ly[p.avg_idx].act_off, y, d.theta, p.P, l.w_off, l.b_off, grad,
                                ctx->at<float>(p.off_dh), loss, C, rmap, B, l.Ci, l.Co, d.label_smoothing, s));
    }
  }

  // backward: head pooling, then every conv from the top down
  {
    const LayerInfo &hc = p.ly[p.head_conv];
    // (with routing codes the head conv's output is not read)
    const double rd = hc.hcode ? 0.25 * hc.Ho * hc.Wo : p.esz * hc.Ho * hc.Wo;
    LAUNCH_T("head_pool_bwd", 0.0, (double)C * B * hc.Co * (rd + p.esz * hc.Ho * hc.Wo + 4.0),
             launch_head_pool_bwd(p.dtype, ws + hc.act_off, ctx->at<float>(p.off_dh), ws + hc.gpre_off, C, rmap, B,
                                  hc.Ho, hc.Wo, hc.Co, p.head_maxpool ? 1 : 0, s,
                                  hc.hcode ? reinterpret_cast<const uint8_t *>(ws + hc.code_off) : nullptr,
                                  hc.act_rs / 4));
  }
  int i = p.head_conv;
  while (i >= 0) {
    const LayerInfo &l = p.ly[i];
    if (l.spec.kind == GCPSL_BLOCK) {
      // the block's gradient at its output sum (gpre, already masked by its
      // ReLU) back through norm2, conv2, norm1, conv1 and the shortcut; the
      // input gradient goes to the layer below, masked by that layer's output
      const BlockInfo &bk = p.blocks[l.blk];
      const LayerInfo &prev = p.ly[i - 1];
      const void *x = input_of(i);
      const char *nn = l.groups ? "groupnorm_bwd" : "batchnorm_bwd";
      const double nby = (double)C * p.esz * B * l.Ho * l.Wo * l.Co * 5.0;
      LAUNCH_T(nn, 0.0, nby, launch_norm_bwd(p.dtype, nargs(bk.n2, ws + bk.c2.act_off, nullptr, ws + l.gpre_off,
                                                             ws + bk.c2.gpre_off, nullptr, 1), s));
      if (int rc = wgrad_run(bk.c2, ws + bk.c2.gpre_off, ws + bk.n1.act_off, 9, l.Co, l.Ho, l.Wo)) return rc;
      if (int rc = conv_dgrad(bk.c2, ws + bk.c2.gpre_off, 9, l.Ho, l.Wo, ws + bk.n1.gpre_off, nullptr,
                              ws + bk.n1.act_off))
        return rc;
      LAUNCH_T(nn, 0.0, nby, launch_norm_bwd(p.dtype, nargs(bk.n1, ws + bk.c1.act_off, nullptr, ws + bk.n1.gpre_off,
                                                             ws + bk.c1.gpre_off, nullptr, 1), s));
      const void *sc_grad = ws + l.gpre_off;  // identity shortcut: the gradient at the sum
      if (bk.proj) {
        LAUNCH_T(nn, 0.0, nby, launch_norm_bwd(p.dtype, nargs(bk.np, ws + bk.cp.act_off, nullptr, ws + l.gpre_off,
                                                               ws + bk.cp.gpre_off, nullptr, 0), s));
        if (int rc = wgrad_run(bk.cp, ws + bk.cp.gpre_off, ws + bk.xs_off, 1, bk.Kcp, l.Ho, l.Wo)) return rc;
        const void *g = ws + bk.cp.gpre_off;
        if (bk.stride == 2) {
          LAUNCH_T("zero_insert", 0.0, (double)C * p.esz * B * l.Co * (l.Ho * l.Wo + (double)l.H * l.W),
                   launch_zero_insert(p.dtype, g, ws + bk.gup_off, C, rmap, B, l.H, l.W, l.Ho, l.Wo, l.Co, s));
          g = ws + bk.gup_off;
        }
        if (int rc = conv_dgrad(bk.cp, g, 1, l.H, l.W, ws + bk.gsc_off, nullptr, nullptr)) return rc;
        sc_grad = ws + bk.gsc_off;
      }
      if (bk.stride == 2) {
        if (int rc = wgrad_run(bk.c1, ws + bk.c1.gpre_off, ws + bk.cols1_off, 1, bk.Kc1, l.Ho, l.Wo)) return rc;
        LAUNCH_T("zero_insert", 0.0, (double)C * p.esz * B * l.Co * (l.Ho * l.Wo + (double)l.H * l.W),
                 launch_zero_insert(p.dtype, ws + bk.c1.gpre_off, ws + bk.gup_off, C, rmap, B, l.H, l.W, l.Ho, l.Wo,
                                    l.Co, s));
        if (int rc = conv_dgrad(bk.c1, ws + bk.gup_off, 9, l.H, l.W, ws + prev.gpre_off, sc_grad, ws + prev.act_off))
          return rc;
      } else {
        if (int rc = wgrad_run(bk.c1, ws + bk.c1.gpre_off, x, 9, l.Ci, l.H, l.W)) return rc;
        if (int rc = conv_dgrad(bk.c1, ws + bk.c1.gpre_off, 9, l.H, l.W, ws + prev.gpre_off, sc_grad,
                                ws + prev.act_off))
          return rc;
      }
      i -= 1;
      continue;
    }
    if (is_norm(l.spec.kind)) {
      // gamma, beta gradients and dL/dz of the conv below (which has no ReLU)
      const double by = (double)C * p.esz * B * l.H * l.W * l.Co * 5.0;
      LAUNCH_T(l.groups ? "groupnorm_bwd" : "batchnorm_bwd", 0.0, by, launch_norm_bwd(p.dtype, norm_args(i), s));
      i -= 1;
      continue;
    }
    // weight and bias gradient
    // the layer's output gradient: gpre, or (routing codes) the next conv's
    // input gradient at the pool's output with the codes
    const void *gsrc = l.pcode ? (const void *)(ws + p.ly[i + 2].gin_off) : (const void *)(ws + l.gpre_off);
    const uint8_t *gcode = l.pcode ? reinterpret_cast<const uint8_t *>(ws + l.code_off) : nullptr;
    const int64_t g_rs = (int64_t)B * l.H * l.W * l.Co / (l.pcode ? 4 : 1);
    WgradArgs w{};
    w.g = gsrc;
    w.gcode = gcode;
    w.x = input_of(i);
    const bool col = i == 0 && p.col0;
    w.Bt = B; w.H = l.H; w.W = l.W; w.Co = l.Co;
    w.Ci = col ? p.Kc : l.Ci;
    w.taps = col ? 1 : 9;
    w.nw = 9 * l.Ci;
    w.g_rs = g_rs;
    w.x_rs = (int64_t)B * l.H * l.W * w.Ci;
    w.C = C;
    w.rmap = rmap;
    w.splits = l.splits;
    w.chunk = l.chunk;
    if (l.splits == 1) {
      w.dw = grad + l.w_off; w.dw_rs = p.P; w.dw_ss = 0;
      w.db = grad + l.b_off; w.db_rs = p.P; w.db_ss = 0;
    } else {  // the layer's own partials, summed by the SGD pass
      w.dw = ctx->at<float>(p.off_part) + l.part_off; w.dw_rs = l.nw; w.dw_ss = (int64_t)p.C * l.nw;
      w.db = ctx->at<float>(p.off_part) + l.dbpart_off; w.db_rs = l.Co; w.db_ss = (int64_t)p.C * l.Co;
    }
    {
      std::string lab;
      const double M = (double)B * l.H * l.W;
      const double fl = 2.0 * C * M * l.Co * 9.0 * l.Ci;
      const double gby = l.pcode ? (p.esz + 1.0) * M / 4 * l.Co : p.esz * M * l.Co;
      const double by = (double)C * (gby + p.esz * M * l.Ci + 4.0 * l.splits * (l.nw + l.Co));
      size_t t_ = tbegin(ctx, s);
      LAUNCH(launch_wgrad(p.dtype, w, s, &lab));
      tend(ctx, s, t_, lab, fl, by);
    }
    if (i == 0) break;
    // input gradient (the cut gradient when layer i-1 is the client's last pool)
    const LayerInfo &prev = p.ly[i - 1];
    const bool through_pool = prev.spec.kind == GCPSL_MAXPOOL2;
    ConvArgs a{};
    a.src = gsrc;
    a.pool_code = const_cast<uint8_t *>(gcode);
    a.wt = ws + l.wd_off;
    a.out = through_pool ? ws + l.gin_off : ws + prev.gpre_off;
    a.bias = nullptr;
    a.res = (l.spec.flags & GCPSL_RESIDUAL) ? a.src : nullptr;
    a.mask = through_pool ? nullptr : (const void *)(ws + prev.act_off);
    a.Bt = B; a.H = l.H; a.W = l.W; a.Csrc = l.Co; a.N = l.Ci; a.K = 9 * l.Co; a.Kp = l.Kdp;
    a.src_rs = g_rs;
    a.wt_rs = (int64_t)l.Ci * l.Kdp;
    a.out_rs = (int64_t)B * l.H * l.W * l.Ci;
    a.bias_rs = 0;
    a.C = C;
    a.rmap = rmap;
    a.epi = EPI_DGRAD;
    a.taps = 9;
    {
      std::string lab;
      const double M = (double)B * l.H * l.W;
      const double fl = 2.0 * C * M * l.Ci * 9.0 * l.Co;
      const double gby = l.pcode ? (p.esz + 1.0) * M / 4 * l.Co : p.esz * M * l.Co;
      const double by = (double)C * (gby + p.esz * ((double)l.Ci * 9 * l.Co +
                                                   M * l.Ci * (1 + (a.res ? 1 : 0) + (a.mask ? 1 : 0))));
      size_t t_ = tbegin(ctx, s);
      LAUNCH(launch_conv(p.dtype, a, s, &lab));
      tend(ctx, s, t_, lab, fl, by);
    }
    if (through_pool) {
      const LayerInfo &pc = p.ly[i - 2];
      if (!pc.pcode)  // (with routing codes the layer below reads gin itself)
      LAUNCH_T("maxpool_bwd", 0.0, 2.25 * p.esz * (double)C * B * pc.Ho * pc.Wo * pc.Co,
               launch_maxpool_bwd(p.dtype, ws + pc.act_off, ws + l.gin_off, ws + pc.gpre_off, C, rmap, B, pc.Ho, pc.Wo,
                                  pc.Co, s));
      i -= 2;
    } else {
      i -= 1;
    }
  }

  // the update, with the split-K sums of the split layers' weight gradients
  // (20 bytes per parameter and the partials)
  LAUNCH_T("sgd", 3.0 * C * p.P, 20.0 * C * p.P + p.sgd_part_bytes,
           launch_sgd_seg(d.theta, d.momentum_buf, grad, ctx->at<float>(p.off_part),
                          reinterpret_cast<const SgdSeg *>(ctx->ws + p.off_sgdseg), (int)p.sgd_segs.size(),
                          p.sgd_blocks, p.sgd_vec, 256 * p.sgd_vec, p.P, C, rmap, d.lr, d.momentum,
                          d.weight_decay, d.nesterov, s));
  ctx->horizon = std::max<int64_t>(ctx->horizon, std::min<int64_t>(step + 1, p.max_steps));
  return GCPSL_OK;
}

int check_staged(gcpsl_ctx *ctx, int64_t step) {
  if (ctx->staged_lo < 0 || step < ctx->staged_lo || step >= ctx->staged_lo + ctx->staged_n)
    return gcpsl_fail(GCPSL_ESTATE, "step " + std::to_string(step) + " has not been sampled");
  return GCPSL_OK;
}

// Whether cluster n takes a local round at this step.
bool takes_round(const gcpsl_ctx *ctx, int64_t step, int n) {
  return ctx->plan.schedule != GCPSL_SCHED_EPOCH || step % ctx->R < ctx->rounds[n];
}

}  // namespace

extern "C" int gcpsl_step(gcpsl_ctx *ctx, int64_t step, float *loss_out, void *stream) {
  gcpsl_clear_error();
  if (!ctx) return gcpsl_fail(GCPSL_EINVAL, "null context");
  if (int rc = check_staged(ctx, step)) return rc;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const Plan &p = ctx->plan;
  if (p.schedule != GCPSL_SCHED_EPOCH) return run_round(ctx, step, nullptr, p.C, loss_out, s);
  int nrep = 0;
  while (nrep < p.C && takes_round(ctx, step, ctx->order[nrep])) ++nrep;
  return run_round(ctx, step, ctx->at<int32_t>(p.off_order), nrep, loss_out, s);
}

extern "C" int gcpsl_step_replica(gcpsl_ctx *ctx, int64_t step, int32_t replica, float *loss_out, void *stream) {
  gcpsl_clear_error();
  if (!ctx) return gcpsl_fail(GCPSL_EINVAL, "null context");
  if (replica < 0 || replica >= ctx->plan.C) return gcpsl_fail(GCPSL_EINVAL, "replica outside [0, C)");
  if (int rc = check_staged(ctx, step)) return rc;
  if (!takes_round(ctx, step, replica))
    return gcpsl_fail(GCPSL_EINVAL, "cluster " + std::to_string(replica) + " waits at step " + std::to_string(step));
  return run_round(ctx, step, ctx->at<int32_t>(ctx->plan.off_ident) + replica, 1, loss_out,
                   reinterpret_cast<hipStream_t>(stream));
}

extern "C" int gcpsl_epoch_rounds(gcpsl_ctx *ctx, int64_t *rounds, int64_t *slots) {
  gcpsl_clear_error();
  if (!ctx || !rounds || !slots) return gcpsl_fail(GCPSL_EINVAL, "null argument");
  std::copy(ctx->rounds.begin(), ctx->rounds.end(), rounds);
  *slots = ctx->R;
  return GCPSL_OK;
}

extern "C" int gcpsl_fuse(gcpsl_ctx *ctx, void *stream) {
  gcpsl_clear_error();
  if (!ctx) return gcpsl_fail(GCPSL_EINVAL, "null context");
  const Plan &p = ctx->plan;
  double W = 0.0;
  std::vector<double> wh(ctx->sizes.size());
  for (size_t n = 0; n < wh.size(); ++n) W += (wh[n] = (double)ctx->sizes[n]);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  LAUNCH_T("fuse", 2.0 * p.C * p.P, 8.0 * p.C * p.P,
           launch_fuse(ctx->desc.theta, ctx->at<double>(p.off_fw), wh.data(), W, p.C, p.P, s));
  // the server normalisation state, with the same weights (Sec. IV-C)
  if (p.S > 0)
    LAUNCH_T("fuse", 2.0 * p.C * p.S, 8.0 * p.C * p.S,
             launch_fuse(ctx->desc.norm_state, ctx->at<double>(p.off_fw), wh.data(), W, p.C, p.S, s));
  ctx->fusion_bytes += 2 * 4 * (int64_t)p.C * (p.P + p.S);
  return GCPSL_OK;
}

extern "C" int gcpsl_fuse_partial(gcpsl_ctx *ctx, double *partial, void *stream) {
  gcpsl_clear_error();
  if (!ctx || !partial) return gcpsl_fail(GCPSL_EINVAL, "null argument");
  if (reinterpret_cast<uintptr_t>(partial) % 8) return gcpsl_fail(GCPSL_EINVAL, "partial must be 8-byte aligned");
  const Plan &p = ctx->plan;
  std::vector<double> wh(ctx->sizes.size());
  for (size_t n = 0; n < wh.size(); ++n) wh[n] = (double)ctx->sizes[n];
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  LAUNCH_T("fuse_partial", 2.0 * p.C * p.P, (4.0 * p.C + 8.0) * p.P,
           launch_fuse_partial(ctx->desc.theta, partial, ctx->at<double>(p.off_fw), wh.data(), p.C, p.P, s));
  if (p.S > 0)
    LAUNCH_T("fuse_partial", 2.0 * p.C * p.S, (4.0 * p.C + 8.0) * p.S,
             launch_fuse_partial(ctx->desc.norm_state, partial + p.P, ctx->at<double>(p.off_fw), wh.data(), p.C,
                                 p.S, s));
  ctx->fusion_bytes += 4 * (int64_t)p.C * (p.P + p.S);  // every replica's state to the fusion point
  return GCPSL_OK;
}

extern "C" int gcpsl_fuse_finalise(gcpsl_ctx *ctx, const double *partial, int64_t W, void *stream) {
  gcpsl_clear_error();
  if (!ctx || !partial) return gcpsl_fail(GCPSL_EINVAL, "null argument");
  if (reinterpret_cast<uintptr_t>(partial) % 8) return gcpsl_fail(GCPSL_EINVAL, "partial must be 8-byte aligned");
  if (W < 1 || W > ((int64_t)1 << 53)) return gcpsl_fail(GCPSL_EINVAL, "W must lie in [1, 2^53]");
  const Plan &p = ctx->plan;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  LAUNCH_T("fuse_finalise", (double)p.P, (8.0 + 4.0 * p.C) * p.P,
           launch_fuse_finalise(ctx->desc.theta, partial, (double)W, p.C, p.P, s));
  if (p.S > 0)
    LAUNCH_T("fuse_finalise", (double)p.S, (8.0 + 4.0 * p.C) * p.S,
             launch_fuse_finalise(ctx->desc.norm_state, partial + p.P, (double)W, p.C, p.S, s));
  ctx->fusion_bytes += 4 * (int64_t)p.C * (p.P + p.S);  // the fused state back to every replica
  return GCPSL_OK;
}

extern "C" int gcpsl_fuse_replicas(float *theta, int32_t C, int64_t P, const int64_t *weights, void *stream) {
  gcpsl_clear_error();
  if (!theta || !weights) return gcpsl_fail(GCPSL_EINVAL, "null argument");
  if (C < 1 || C > kMaxArgWeights) return gcpsl_fail(GCPSL_EINVAL, "C must lie in [1, 64]");
  if (P < 1) return gcpsl_fail(GCPSL_EINVAL, "P must be >= 1");
  if (reinterpret_cast<uintptr_t>(theta) % 4) return gcpsl_fail(GCPSL_EINVAL, "theta must be 4-byte aligned");
  double wh[kMaxArgWeights];
  double W = 0.0;
  for (int n = 0; n < C; ++n) {
    if (weights[n] < 0 || weights[n] > (int64_t)1 << 29) return gcpsl_fail(GCPSL_EINVAL, "weights must lie in [0, 2^29]");
    W += (wh[n] = (double)weights[n]);
  }
  if (!(W > 0.0)) return gcpsl_fail(GCPSL_EINVAL, "the weights sum to zero");
  HIP_TRY(launch_fuse(theta, nullptr, wh, W, C, P, reinterpret_cast<hipStream_t>(stream)));
  return GCPSL_OK;
}

extern "C" int gcpsl_timing(gcpsl_ctx *ctx, int32_t on) {
  gcpsl_clear_error();
  if (!ctx) return gcpsl_fail(GCPSL_EINVAL, "null context");
  ctx->timing = on != 0;
  return GCPSL_OK;
}

extern "C" int gcpsl_timing_read(gcpsl_ctx *ctx, gcpsl_kernel_stat *out, int32_t cap, int32_t *n) {
  gcpsl_clear_error();
  if (!ctx || !n || (cap > 0 && !out)) return gcpsl_fail(GCPSL_EINVAL, "null argument");
  HIP_TRY(hipDeviceSynchronize());
  std::vector<gcpsl_kernel_stat> agg;
  for (const KernelRec &r : ctx->recs) {
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, ctx->events[r.ev], ctx->events[r.ev + 1]));
    size_t k = 0;
    while (k < agg.size() && r.name != agg[k].name) ++k;
    if (k == agg.size()) {
      gcpsl_kernel_stat st{};
      std::snprintf(st.name, sizeof(st.name), "%s", r.name.c_str());
      agg.push_back(st);
    }
    agg[k].launches += 1;
    agg[k].ms += ms;
    agg[k].flops += r.flops;
    agg[k].bytes += r.bytes;
  }
  ctx->recs.clear();
  ctx->next_event = 0;
  *n = (int32_t)agg.size();
  for (int32_t k = 0; k < cap && k < (int32_t)agg.size(); ++k) out[k] = agg[k];
  return GCPSL_OK;
}

extern "C" int gcpsl_participation(gcpsl_ctx *ctx, int64_t *active_slots, int64_t *total_slots, int32_t *per_step) {
  gcpsl_clear_error();
  if (!ctx || !active_slots || !total_slots) return gcpsl_fail(GCPSL_EINVAL, "null argument");
  const Plan &p = ctx->plan;
  HIP_TRY(hipDeviceSynchronize());
  const int64_t T = ctx->horizon;
  std::vector<int32_t> hits((size_t)std::max<int64_t>(T, 1) * p.C, 0);
  if (T > 0) HIP_TRY(hipMemcpy(hits.data(), ctx->ws + p.off_hits, sizeof(int32_t) * T * p.C, hipMemcpyDeviceToHost));
  int64_t act = 0;
  for (int64_t i = 0; i < T * p.C; ++i) act += hits[i];
  *active_slots = act;
  *total_slots = (int64_t)p.K * T;
  if (per_step && T > 0) std::copy(hits.begin(), hits.begin() + T * p.C, per_step);
  return GCPSL_OK;
}

extern "C" int gcpsl_batch_deviation(gcpsl_ctx *ctx, int64_t *sum_num, int64_t *batches, int64_t *denom,
                                     int64_t *per_step) {
  gcpsl_clear_error();
  if (!ctx || !sum_num || !batches || !denom) return gcpsl_fail(GCPSL_EINVAL, "null argument");
  const Plan &p = ctx->plan;
  HIP_TRY(hipDeviceSynchronize());
  const int64_t T = ctx->horizon;
  std::vector<int64_t> dev((size_t)std::max<int64_t>(T, 1) * p.C, -1);
  if (T > 0) HIP_TRY(hipMemcpy(dev.data(), ctx->ws + p.off_dev, sizeof(int64_t) * T * p.C, hipMemcpyDeviceToHost));
  int64_t sum = 0, cnt = 0;
  for (int64_t i = 0; i < T * p.C; ++i)
    if (dev[i] >= 0) {
      sum += dev[i];
      cnt += 1;
    }
  *sum_num = sum;
  *batches = cnt;
  *denom = (int64_t)p.B * p.n_examples;
  if (per_step && T > 0) std::copy(dev.begin(), dev.begin() + T * p.C, per_step);
  return GCPSL_OK;
}

extern "C" int gcpsl_payload(gcpsl_ctx *ctx, int64_t *bytes) {
  gcpsl_clear_error();
  if (!ctx || !bytes) return gcpsl_fail(GCPSL_EINVAL, "null argument");
  const Plan &p = ctx->plan;
  HIP_TRY(hipDeviceSynchronize());
  const int64_t T = ctx->horizon;
  std::vector<int32_t> hits((size_t)std::max<int64_t>(T, 1) * p.C, 0);
  if (T > 0) HIP_TRY(hipMemcpy(hits.data(), ctx->ws + p.off_hits, sizeof(int32_t) * T * p.C, hipMemcpyDeviceToHost));
  const LayerInfo &cl = p.ly[p.cut - 1];
  const int64_t cut_bytes = (int64_t)cl.Ho * cl.Wo * cl.Co * p.esz;  // one example's cut activation
  int64_t act = 0, cg = 0, up = 0, down = 0;
  for (int64_t t = 0; t < T; ++t)
    for (int n = 0; n < p.C; ++n) {
      if (!takes_round(ctx, t, n)) continue;
      act += (int64_t)p.B * (cut_bytes + 4);  // activations and labels, client -> server
      cg += (int64_t)p.B * cut_bytes;         // cut gradients, server -> client
      up += (int64_t)hits[t * p.C + n] * p.Pc * 4;
      down += ctx->clients_in[n] * p.Pc * 4;
    }
  bytes[GCPSL_PAYLOAD_ACTIVATIONS] = act;
  bytes[GCPSL_PAYLOAD_CUT_GRADS] = cg;
  bytes[GCPSL_PAYLOAD_CLIENT_GRADS] = up;
  bytes[GCPSL_PAYLOAD_CLIENT_MODEL] = down;
  bytes[GCPSL_PAYLOAD_FUSION] = ctx->fusion_bytes;
  return GCPSL_OK;
}

extern "C" int gcpsl_tensor(gcpsl_ctx *ctx, const char *name, void **ptr, int64_t *numel, int32_t *dtype) {
  gcpsl_clear_error();
  if (!ctx || !name || !ptr || !numel || !dtype) return gcpsl_fail(GCPSL_EINVAL, "null argument");
  const Plan &p = ctx->plan;
  const std::string nm(name);
  const int64_t CB = (int64_t)p.C * p.B;
  auto put = [&](size_t off, int64_t ne, int32_t dt) {
    *ptr = ctx->ws + off;
    *numel = ne;
    *dtype = dt;
    return GCPSL_OK;
  };
  if (nm == "x") return put(p.off_x, (int64_t)p.max_window * p.x_rs, p.dtype);
  if (nm == "idx") return put(p.off_idx, (int64_t)p.max_window * CB, -1);
  if (nm == "y") return put(p.off_y, (int64_t)p.max_window * CB, -1);
  if (nm == "hits") return put(p.off_hits, p.max_steps * p.C, -1);
  if (nm == "dh") return put(p.off_dh, CB * p.Ch_head, GCPSL_F32);
  if (nm == "grad") return put(p.off_grad, (int64_t)p.C * p.P, GCPSL_F32);
  for (size_t i = 0; i < p.ly.size(); ++i) {
    const LayerInfo &l = p.ly[i];
    const std::string k = std::to_string(i);
    if (l.spec.kind == GCPSL_BLOCK) {
      // internals of block i: conv outputs z<i>.1 .2 .p, norm1 output
      // act<i>.n1, shortcut sc<i>; gradients dz<i>.1 .2 .p (conv outputs),
      // gpre<i>.n1 (norm1), gpre<i> (the block's output sum), gsc<i> (the
      // shortcut's input gradient)
      const BlockInfo &bk = p.blocks[l.blk];
      const int64_t rs = (int64_t)p.C * l.act_rs, rs_in = (int64_t)p.C * p.B * l.H * l.W * l.Ci;
      if (nm == "act" + k) return put(l.act_off, rs, p.dtype);
      if (nm == "gpre" + k) return put(l.gpre_off, rs, p.dtype);
      if (nm == "z" + k + ".1") return put(bk.c1.act_off, rs, p.dtype);
      if (nm == "z" + k + ".2") return put(bk.c2.act_off, rs, p.dtype);
      if (nm == "act" + k + ".n1") return put(bk.n1.act_off, rs, p.dtype);
      if (nm == "dz" + k + ".1") return put(bk.c1.gpre_off, rs, p.dtype);
      if (nm == "dz" + k + ".2") return put(bk.c2.gpre_off, rs, p.dtype);
      if (nm == "gpre" + k + ".n1") return put(bk.n1.gpre_off, rs, p.dtype);
      if (bk.proj && nm == "z" + k + ".p") return put(bk.cp.act_off, rs, p.dtype);
      if (bk.proj && nm == "sc" + k) return put(bk.np.act_off, rs, p.dtype);
      if (bk.proj && nm == "dz" + k + ".p") return put(bk.cp.gpre_off, rs, p.dtype);
      if (bk.proj && nm == "gsc" + k) return put(bk.gsc_off, rs_in, p.dtype);
      continue;
    }
    if (nm == "act" + k && l.stored) return put(l.act_off, (int64_t)p.C * l.act_rs, p.dtype);
    if ((l.pcode || l.hcode) && nm == "route" + std::to_string(i + 1))
      return put(l.code_off, (int64_t)p.C * l.act_rs / 4, -2);
    if (l.spec.kind == GCPSL_CONV3X3 || is_norm(l.spec.kind)) {
      const int64_t rs = (int64_t)p.B * l.H * l.W;
      if (nm == "gpre" + k && !l.pcode) return put(l.gpre_off, p.C * rs * l.Co, p.dtype);
      if (nm == "gin" + k && l.has_gin) return put(l.gin_off, p.C * rs * l.Ci, p.dtype);
    }
  }
  return gcpsl_fail(GCPSL_EINVAL, "unknown tensor " + nm);
}
