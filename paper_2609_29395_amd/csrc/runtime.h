// Host runtime internals: error state, the layer plan and kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <string>
#include <vector>

#include "../../include/gcpsl.h"
#include "common.h"

// One-time set-up that belongs to a device (kernel attributes such as the
// dynamic LDS limit): bit d records device d; a device id past 31 (or a
// failed query) repeats the set-up on every call, which is harmless.
struct PerDeviceOnce {
  std::atomic<uint32_t> done{0};
  static int current() {
    int d = -1;
    return hipGetDevice(&d) == hipSuccess ? d : -1;
  }
  bool needed() const {
    const int d = current();
    return d < 0 || d >= 32 || (done.load(std::memory_order_acquire) & (1u << d)) == 0;
  }
  void mark() {
    const int d = current();
    if (d >= 0 && d < 32) done.fetch_or(1u << d, std::memory_order_acq_rel);
  }
};

// ----------------------------------------------------------------- errors
void gcpsl_clear_error();
int gcpsl_fail(int code, const std::string &msg);

// ------------------------------------------------------------ kernel args

// Implicit-GEMM 3x3 conv, forward or input-gradient form:
//   out[m][n] = epi( sum_k A[m][k] * Wt[n][k] ),  m = (b, h, w), k = (r, s, c)
//   A[m][k] = src[b][h + r - 1][w + s - 1][c] (zero outside the image).
enum ConvEpi { EPI_FWD = 0, EPI_DGRAD = 1 };
struct ConvArgs {
  const void *src;   // [C][Bt][H][W][Csrc]
  const void *wt;    // [C][N][Kp]  (k = (r, s, c), rows zero-padded to Kp)
  void *out;         // [C][Bt][H][W][N]
  const float *bias; // fwd: [C][...] bias of this layer (stride bias_rs)
  const void *res;   // residual input [C][Bt][H][W][N] or null
  const void *mask;  // dgrad: mask source [C][Bt][H][W][N] (value > 0) or null
  int Bt, H, W, Csrc, N, K, Kp;
  int64_t src_rs, wt_rs, out_rs, bias_rs;  // per-replica strides (elements)
  int C;     // replica slots of the launch
  int pool_max;  // with the per-image mean in pool_out: the mean of the 2x2 max pool (in the padding
                 // after C, so no other field moves)
  const int32_t *rmap;  // device [C]: replica of each slot, or null (slot z = replica z)
  int epi;
  int taps;  // 9: 3x3 implicit GEMM; 1: src already holds im2col rows, A[m][k] = src[m][k]
  int res_lds;  // set by the launcher: the residual (== src) is taken from the staged centre tap
  int no_relu;  // fwd: store the raw output (a norm layer follows)
  void *pool_out;      // fwd: also a pooling of the output, else null: the 2x2 max pool
                       // [C][Bt][H/2][W/2][N] (kernels that report conv_fuses_pool) or the mean over
                       // each image's positions, of the 2x2 max pool if pool_max, [C][Bt][N] (kernels
                       // that report conv_fuses_avg)
  int64_t pool_rs;     // its per-replica stride (elements)
  // Routing codes of a 2 x 2 max pool, one byte per pooled element: 0..3 =
  // the window position (row-major) of the first maximum, 4 = no gradient
  // (the maximum is not positive, so the ReLU below it is off).  fwd (with
  // the max pool in pool_out, kernels that report conv_pool_codes): written
  // beside pool_out in its layout, and `out` is then not written.  dgrad: src
  // holds the pooled gradient [C][Bt][H/2][W/2][Csrc] (stride src_rs) and the
  // kernel routes it to the unpooled grid through these codes (same layout).
  uint8_t *pool_code;
  int64_t code_rs;  // fwd with the head's mean of a max pool in pool_out (kernels that report
                    // conv_fuses_avg): the pool's routing codes [C][Bt][H/2][W/2][N] go to
                    // pool_code, this its per-replica stride, and `out` is not written
};

// Weight gradient: dW[co][kk] = sum_p G[p][co] X(p, kk), kk = (r, s, ci),
// and (optionally) db[co] = sum_p G[p][co].  Split over pixel ranges.
struct WgradArgs {
  const void *g;  // [C][Bt][H][W][Co] pre-activation gradient
  const void *x;  // [C][Bt][H][W][Ci] layer input
  float *dw;      // split s, replica r: dw + s*dw_ss + r*dw_rs, [Co][9Ci]
  float *db;      // db + s*db_ss + r*db_rs, [Co]
  int Bt, H, W, Ci, Co;
  int64_t g_rs, x_rs, dw_rs, dw_ss, db_rs, db_ss;
  int C, splits, chunk;  // replica slots; pixel chunk per split (multiple of the k tile)
  const int32_t *rmap;   // device [C]: replica of each slot, or null (slot z = replica z)
  int taps;  // 9: x is the layer input; 1: x holds im2col rows of Ci columns
  int nw;    // weight-gradient row length written (9 * input channels)
  // or null; else g holds the gradient at the output of the 2 x 2 max pool
  // after this layer, [C][Bt][H/2][W/2][Co] (stride g_rs), and gcode its
  // routing codes (ConvArgs::pool_code): the pre-activation gradient is
  // g routed through them (kernels that report wgrad_pool_codes)
  const uint8_t *gcode;
};

// ---------------------------------------------------------------- launchers
// label (optional) receives the kernel instantiation chosen for the shape.
hipError_t launch_conv(int dtype, const ConvArgs &a, hipStream_t s, std::string *label = nullptr);
hipError_t launch_wgrad(int dtype, const WgradArgs &a, hipStream_t s, std::string *label = nullptr);
int wgrad_k_tile(int dtype);
// bf16 weight gradient with LDS-direct tile copies and transposing LDS reads
// (k_wgrad_lds.hip): usable when wgrad_lds_ok; needs chunk % 64 == 0.
bool wgrad_lds_ok(int dtype, int Co, int Ci);
// the image layer's weight gradient on its im2col rows (32 channels, 32 columns)
bool wgrad_col_ok(int dtype, int Co, int Ci, int taps);
hipError_t launch_wgrad_col(const WgradArgs &a, hipStream_t s, std::string *label);
void wgrad_lds_tile(int Co, int Ci, int H, int W, int taps, int *bm, int *bn, int *bk, int *per_cu);
hipError_t launch_wgrad_lds(const WgradArgs &a, hipStream_t s, std::string *label);
// bf16 forward / dgrad of 32 x 32 image layers with 32 or 64 channels
// (k_conv_img.hip): one halo-staged 8-row tile and the whole weight matrix
// per workgroup.
bool conv_img_ok(int dtype, const ConvArgs &a);
// the image layer's forward on its im2col rows (32 columns, 32 channels)
bool conv_col_ok(int dtype, const ConvArgs &a);
// the image layer on the bf16 NHWC images themselves (3 -> 32 channels,
// 32-pixel-wide images, a multiple of 8 rows): forward and weight gradient
// build its im2col rows in LDS
bool conv_im3_ok(int dtype, int Ci, int Co, int H, int W);
hipError_t launch_conv_col(const ConvArgs &a, hipStream_t s, std::string *label);
// whether launch_conv also writes ConvArgs::pool_out for this layer
bool conv_fuses_pool(int dtype, const ConvArgs &a);
// whether launch_conv takes ConvArgs::pool_code for these arguments (fwd:
// writes the codes with the pool instead of the unpooled output; dgrad: a
// pooled source routed through them)
bool conv_pool_codes(int dtype, const ConvArgs &a);
// whether launch_wgrad takes WgradArgs::gcode for this layer shape
bool wgrad_pool_codes(int dtype, int Co, int Ci, int H, int W, int taps);
// Whether launch_conv writes the per-image mean (of the 2x2 max pool if
// pool_max) to pool_out for these arguments (16 x 16 bf16 images on the
// 256-wide halo tile, every output channel in one tile).
bool conv_fuses_avg(int dtype, const ConvArgs &a);
hipError_t launch_conv_img(const ConvArgs &a, hipStream_t s, std::string *label);
// bf16 forward / dgrad with LDS-direct tile copies (k_conv_lds.hip).
bool conv_lds_ok(int dtype, const ConvArgs &a);
hipError_t launch_conv_lds(const ConvArgs &a, hipStream_t s, std::string *label);
// Workgroup tile (rows = output channels, cols = 9 * input channels) the
// weight-gradient launcher uses for a layer; the split-K plan depends on it.
void wgrad_tile(int dtype, int Co, int ncols, int *bm, int *bn);

// Largest L the sampler's batch-deviation histogram holds (LDS, Sec. V-E).
constexpr int kMaxDevClasses = 4096;
hipError_t launch_sample(const int32_t *ids, const int64_t *off, const int32_t *coe,
                         const int32_t *labels, const int64_t *ghist, int32_t *idx, int32_t *y, int32_t *hits,
                         int64_t *dev, int C, int B, int K, int L, int64_t nex, uint64_t seed, int64_t step0,
                         int nsteps, int64_t max_steps, int64_t R, hipStream_t s);
hipError_t launch_gather(const float *images, const int32_t *idx, void *x, int dtype,
                         int64_t rows, int64_t row_elems, hipStream_t s);
// Gather with im2col: x[row][pixel][k], k = (r, s, c) < 9 Cin, zero to Kc.
hipError_t launch_gather_im2col(const float *images, const int32_t *idx, void *x, int dtype,
                                int64_t rows, int H, int W, int Cin, int Kc, hipStream_t s);
// Compute copies of every conv layer's weights in one launch: per layer a
// forward copy wf [C][co][Kp] (one workgroup per output row) and, except for
// the image layer, an input-gradient copy wd [C][ci][Kdp] (one workgroup per
// 64 x 64 block and kernel tap).
struct PrepJob {
  int64_t w_off;  // the layer's weights in a replica's parameter vector
  void *dst;      // wf or wd of replica 0 (replica r at r * co * kpad / r * ci * kpad)
  int co, ci, kpad;
  int kind;   // 0 forward copy, 1 input-gradient copy, 2 both (dst = wd, dst2 = wf)
  int first;  // first workgroup of the job
  void *dst2 = nullptr;  // kind 2: wf
  int kpad2 = 0;         // kind 2: Kp
  int taps = 9;          // kernel taps: 9 (3 x 3) or 1 (1 x 1)
};
constexpr int kMaxPrepJobs = 48;
struct PrepJobs {
  PrepJob j[kMaxPrepJobs];
  int n = 0, total = 0;  // jobs, workgroups per replica
};
// Appends the jobs of one layer (wd may be null) with 9 (3 x 3) or 1 (1 x 1)
// kernel taps.
void prep_add_layer(PrepJobs &jobs, int64_t w_off, int co, int ci, void *wf, int Kp, void *wd, int Kdp,
                    int taps = 9);
hipError_t launch_prep_weights(int dtype, const float *theta, int64_t P, int C, const int32_t *rmap,
                               const PrepJobs &jobs, hipStream_t s);
hipError_t launch_maxpool_fwd(int dtype, const void *x, void *z, int C, const int32_t *rmap, int Bt, int H, int W,
                              int Ch, hipStream_t s);
hipError_t launch_maxpool_bwd(int dtype, const void *a, const void *gz, void *gpre, int C, const int32_t *rmap,
                              int Bt, int H, int W, int Ch, hipStream_t s);
hipError_t launch_head_pool(int dtype, const void *a, void *h, int C, const int32_t *rmap, int Bt, int H, int W,
                            int Ch, int maxpool, hipStream_t s);
// LDS the classifier-head kernel stages (pooled features, weights, logits).
constexpr size_t kMaxLinearLds = 160 * 1024;
inline size_t linear_ce_lds_bytes(int Bt, int Ch, int L) {
  return sizeof(float) * ((size_t)Bt * (Ch + 1) + (size_t)L * (Ch + 1) + (size_t)Bt * L + Bt + L);
}
// Register-resident head (weights in registers, one 4-channel slice per
// lane): heads of at most 256 channels (a multiple of 4) and kHeadRegL
// classes, on kHeadRegWaves waves; its LDS holds the logits, the per-example
// losses and the weight-gradient hand-over of the reduction tree.
constexpr int kHeadRegL = 16, kHeadRegWaves = 8;
inline size_t linear_ce_reg_lds_bytes(int Bt, int L) {
  return sizeof(float) * ((((size_t)Bt * (L + 1) + 3) & ~(size_t)3) + (size_t)(kHeadRegWaves / 2) * L * 64 * 4);
}
inline bool linear_ce_reg_ok(int Bt, int Ch, int L) {
  return Ch % 4 == 0 && Ch <= 256 && L <= kHeadRegL && linear_ce_reg_lds_bytes(Bt, L) <= kMaxLinearLds;
}
// The classifier head (linear layer and softmax cross-entropy, one workgroup
// per replica): the register-resident kernel where linear_ce_reg_ok holds,
// else the LDS-staged one.
hipError_t launch_linear_ce(int dtype, const void *h, const int32_t *y, const float *theta,
                            int64_t P, int64_t w_off, int64_t b_off, float *grad, float *dh,
                            float *loss, int C, const int32_t *rmap, int Bt, int Ch, int L, float eps,
                            hipStream_t s);
// maxpool with code (bf16, the head conv's routing codes [C][Bt][H/2][W/2][Ch],
// per-replica stride code_rs): the gradient is routed through the codes and
// `a` is not read
hipError_t launch_head_pool_bwd(int dtype, const void *a, const float *dh, void *gpre, int C, const int32_t *rmap,
                                int Bt, int H, int W, int Ch, int maxpool, hipStream_t s,
                                const uint8_t *code = nullptr, int64_t code_rs = 0);
// SGD on the replicas of the launch's slots: P parameters each, row stride P.
// SGD over the parameter vector in segments: a segment [begin, begin + len)
// takes its gradient from grad (splits = 0) or is the ordered sum of
// `splits` split-K partials, element j of split k for replica r at
// partials[src + k ss + r rs + j], which is also written to grad.  Blocks of
// kSgdBlockElems elements, or split_elems in a segment of partials (one
// vector per thread, so that the partial loads spread over enough blocks);
// a segment's blocks start at first_block.
struct SgdSeg {
  int64_t begin, len, src, ss, rs;
  int32_t splits, first_block;
};
constexpr int kSgdBlockElems = 4096;
hipError_t launch_sgd_seg(float *theta, float *mom, float *grad, const float *partials, const SgdSeg *segs, int nseg,
                          int blocks, int vec, int split_elems, int64_t P, int C, const int32_t *rmap, float lr,
                          float mu, float wd, int nesterov, hipStream_t s);
// Eq. 5 over C replicas of P parameters: weights from w_host through the
// kernel arguments when C <= kMaxArgWeights, else from w_dev (device).
constexpr int kMaxArgWeights = 64;
hipError_t launch_fuse(float *theta, const double *w_dev, const double *w_host, double W, int C, int64_t P,
                       hipStream_t s);
// The fusion in two halves (fp64 partial sum to a buffer, then division,
// rounding and broadcast); the same result as launch_fuse bit for bit.
hipError_t launch_fuse_partial(const float *theta, double *partial, const double *w_dev, const double *w_host,
                               int C, int64_t P, hipStream_t s);
hipError_t launch_fuse_finalise(float *theta, const double *partial, double W, int C, int64_t P, hipStream_t s);

// Normalisation layers (k_norm.hip): batch norm (groups == 0) or group norm
// over a conv's raw output z, followed by ReLU.
struct NormArgs {
  const void *z;  // [C][Bt*H*W][Ch] raw conv output, replica stride z_rs
  void *a;        // forward output a = ReLU(gamma x_hat + beta), stride z_rs
  const void *du; // backward: dL/du (ReLU-masked), stride z_rs
  void *dz;       // backward: dL/dz, stride z_rs
  float *mean, *rstd;  // [C][nstat] statistics (per channel, or per example and group)
  double *part;        // [C][chunks][Ch][2] per-chunk channel sums
  double *sums;        // [C][nstat][2] sums for the input gradient
  const float *theta;  // [C][P] parameters (gamma at g_off, beta at b_off)
  float *grad;         // [C][P] gradient (dgamma, dbeta written)
  float *state;        // [C][S] normalisation state (batch norm: running mean, var, counter at st_off)
  int64_t P, g_off, b_off, S, st_off, z_rs;
  int Bt, H, W, Ch, groups, nstat;
  int chunks, chunk_px;  // pixel chunks of the channel reductions
  int C;                 // replica slots
  const int32_t *rmap;   // device [C]: replica of each slot, or null
  const void *res = nullptr;  // forward: added to gamma x_hat + beta before the ReLU (a block's shortcut), or null
  int relu = 1;               // forward: 1 applies the ReLU, 0 stores gamma x_hat + beta (a shortcut's norm)
};
bool norm_ok(int dtype, int Ch, int groups);
// Operand staging of a block's strided convolutions (k_block.hip).
hipError_t launch_im2col(int dtype, const void *x, void *cols, int C, const int32_t *rmap, int Bt, int H, int W,
                         int Ci, int Ho, int Wo, int R, int S, int stride, int pad, int Kc, hipStream_t s);
hipError_t launch_zero_insert(int dtype, const void *g, void *gup, int C, const int32_t *rmap, int Bt, int H, int W,
                              int Ho, int Wo, int Ch, hipStream_t s);
hipError_t launch_norm_fwd(int dtype, const NormArgs &a, hipStream_t s);
hipError_t launch_norm_bwd(int dtype, const NormArgs &a, hipStream_t s);
