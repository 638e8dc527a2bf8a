// Host-side launch interface between the C ABI layer and the gfx950 kernels.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace numbat {

constexpr int kMaxTaps = 25;

// Kernel classes for the optional launch timing (numbat_timing_*).  A launcher names the
// class of its kernels with trace_begin / trace_end around their launches.  While timing
// is enabled, every launch made through NUMBAT_LAUNCH carries a start and a stop event
// that take the dispatch's own begin and end timestamps (hipExtLaunchKernelGGL), so a
// class's time is its kernels' execution time alone, without launch gaps or the time an
// event marker of its own would add; with timing off it is a plain hipLaunchKernelGGL.
enum KernelClass {
  KC_CONV_FWD = 0,      // implicit GEMM, forward
  KC_STATS_MERGE,       // batch statistics merge
  KC_DGRAD_WEIGHTS,     // data-gradient weight re-layout
  KC_CONV_DGRAD,        // implicit GEMM, data-gradient phases
  KC_WGRAD,             // weight-gradient GEMM
  KC_SPLITK_REDUCE,     // weight-gradient split reduction
  KC_BN_STATS,          // standalone BN statistics
  KC_BN_FWD,            // BN + SiLU forward apply
  KC_BN_BWD_REDUCE,     // BN + SiLU backward reduce
  KC_BN_BWD_FINALIZE,   // BN + SiLU backward finalize
  KC_BN_BWD_APPLY,      // BN + SiLU backward apply
  KC_PACK,              // 8-channel repacking of a 3-channel image input
  KC_OPT_SUMSQ,         // optimiser step: squared-norm partials of the gradients
  KC_OPT_UPDATE,        // optimiser step: clipped SGD-Nesterov update
  KC_POOL,              // SPPF max pool and neck upsampling, forward and backward
  KC_COUNT
};
void trace_begin(int cls);
void trace_end(int cls);
// a start / stop event pair for the next launch, recorded under the current class; false
// when timing is off (or no class is open, or no event could be created)
bool timing_events(hipEvent_t* start, hipEvent_t* stop);

#define NUMBAT_LAUNCH(kernel, grid, block, smem, stream, ...)                                        \
  do {                                                                                               \
    hipEvent_t numbat_ev0_, numbat_ev1_;                                                             \
    if (::numbat::timing_events(&numbat_ev0_, &numbat_ev1_))                                         \
      hipExtLaunchKernelGGL(kernel, grid, block, smem, stream, numbat_ev0_, numbat_ev1_, 0, __VA_ARGS__); \
    else                                                                                             \
      hipLaunchKernelGGL(kernel, grid, block, smem, stream, __VA_ARGS__);                           \
  } while (0)

// conv GEMM kernel variants: generic (source channels a multiple of 8; A fragments loaded
// into registers), and the direct-to-LDS kernel for 16-multiple channel counts of at least
// 32 in its stage configurations (three or two stages, 32- or 64-element steps, four or
// eight waves)
enum { kVariantGeneric = 0, kVariantDma3 = 3, kVariantDma2 = 4, kVariantDma32 = 5, kVariantDma3W8 = 7, kVariantHalo = 11 };
struct TileCfg {
  int bm, bn;
  int id;       // instantiation id
  int variant;  // kVariant*
};

// Implicit GEMM (conv_gemm.hip) D[M][N] = A[M][K] * B[N][K]^T for source channel
// counts that are multiples of 8:
//   row m   = (img, gi, gj) on a gh x gw grid per image,
//   k       = (tap, c), c < cs, K = taps * cs,
//   A[m][k] = src[img, gi*gstride_h + off_h[tap], gj*gstride_w + off_w[tap], c]  (0 outside hs x ws),
//   B[n][k] = wt[n * ktot + k]   (K-major), or with bt set (the data gradient's weights
//             read in place): k = (tap, o), o < cs, B[n][k] = wt[o * wostep/2 + tap offset + n]
// D written (bf16) to dst[img, gi*dstep_h + doff_h, gj*dstep_w + doff_w, n].  The forward
// convolution is one such GEMM; the stride phases of a data gradient are up to four
// "phases" sharing one launch (blockIdx.z), each with its own grid, taps, offsets, B
// matrix and destination offset.
//
// The taps of every phase form a grid (rows of tw taps; off_h and off_w change by a
// constant +-1 from column to column and row to row).  convgemm_launch derives from
// off[] the byte steps the 16-channel fast path walks the taps with (tw, toff0, cstep,
// rstep, halo_px); callers fill in off[] only.
constexpr int kMaxPhases = 4;
struct GemmPhase {
  const bf16_t* wt;     // [nout][ktot], K-major
  int32_t taps, ktot;   // ktot = taps * cs
  int32_t gh, gw, m;    // m = nimg * gh * gw
  FastDiv div_gw, div_ghw;
  int32_t doff_h, doff_w;
  int32_t off[kMaxTaps];  // (off_h & 0xffff) | (off_w << 16)
  // set by convgemm_launch: taps per grid row, byte offset of tap 0 (plus the halo
  // shift), byte step to the next tap in a row and from a row's last tap to the next
  // row's first; grid rows, offsets of tap 0 and the (+-1 or 0) offset steps between
  // grid rows and columns
  int32_t tw, toff0, cstep, rstep;
  int32_t th, dh0, dw0, tsh, tsw;
  // transposed B (bt): byte offset of tap 0's weights, byte step per o, byte steps to the
  // next tap in a grid row and from a row's last tap to the next row's first
  int32_t wtoff0, wostep, wcstep, wrstep;
};
struct ConvGemmArgs {
  const bf16_t* src;
  int64_t src_pix;
  int32_t hs, ws, cs;
  int32_t nout, nimg;
  int32_t gstride_h, gstride_w;
  bf16_t* dst;
  int64_t dst_pix;
  int32_t hd, wd, dstep_h, dstep_w;
  int32_t accumulate;
  float2* stats_part;  // phase 0 only: [m tiles][nout] (tile mean, tile M2) or nullptr
  int32_t nphase;
  int32_t halo_px;     // set by convgemm_launch: pixels the fast path's gather base sits before an image
  int32_t remap;       // set by convgemm_launch: XCD-aware tile order (see xcd_remap)
  int32_t bt;          // B is the OHWI weight tensor read in place (direct-to-LDS kernel only)
  // epilogue operation on each fp32 result before rounding (inference paths; never with
  // accumulate or statistics): kPostNone, kPostBias (+ bias[n]) or kPostBnSilu
  // (SiLU(gamma (v - mean) / sqrt(var + eps) + beta) with running statistics)
  int32_t post;
  float post_eps;
  const float* post_bias;
  const float *post_gamma, *post_beta, *post_mean, *post_var;
  // prologue (halo kernel), pro_kind:
  //  kProNone
  //  kProFwd (forward): the source is the previous layer's pre-BN output, and its BN (batch
  //    statistics pro_mean / pro_var, pro_gamma, pro_beta, pro_eps) + SiLU is applied to the
  //    staged halo before the taps read it
  //  kProBwd (data gradient): the source is g = dL/d(activation) of this layer's BN + SiLU,
  //    and the staged halo becomes dy = that backward of (g, pro_y) with the batch statistics
  //    pro_mean / pro_rstd, pro_gamma, pro_beta and the reduced pro_dgamma / pro_dbeta over
  //    pro_m rows; dy of every tile's own pixels is also written to pro_dy (the first column
  //    tile's blocks write it)
  int32_t pro_kind;
  const float *pro_gamma, *pro_beta, *pro_mean, *pro_var;
  float pro_eps;
  const float *pro_rstd, *pro_dgamma, *pro_dbeta;
  const bf16_t* pro_y;
  bf16_t* pro_dy;
  int64_t pro_y_pix, pro_dy_pix, pro_m;
  GemmPhase ph[kMaxPhases];
};
enum { kProNone = 0, kProFwd = 1, kProBwd = 2 };
constexpr int kProMaxC = 1024;  // most source channels the prologue stages constants for
enum { kPostNone = 0, kPostBias = 1, kPostBnSilu = 2 };
// tile and kernel for a problem with at most m_max rows per phase, nout columns, cs
// source channels, reduction length ktot and nphase phases; bt: the weights are read in
// place (transposed B) if the direct-to-LDS kernel takes the problem
TileCfg convgemm_pick(int64_t m_max, int nout, int cs, int ktot, int nphase, bool bt);
// a is taken by value: the launcher completes the tap-walk fields
hipError_t convgemm_launch(ConvGemmArgs a, const TileCfg& t, hipStream_t s, int cls);
// whether the direct-to-LDS kernel takes the problem on tile t (it can read B in place)
bool convgemm_direct(ConvGemmArgs a, const TileCfg& t);
// 3x3, stride-1, padding-1 convolutions whose input halo is staged in LDS once per
// 32-channel chunk (conv_gemm.hip, convhalo_kernel): the forward (K-major weights, taps in
// off[]) and the data gradient (bt: the OHWI weights read in place, flipped; off[] unused).
// convhalo_shape: whether the kernel takes the problem; convhalo_pick: its tile for m rows,
// nout columns and an h x w image, bt for the data gradient, any_grid to take small forward
// grids too (variant kVariantGeneric when the halo kernel is not the one to use).
bool convhalo_shape(const ConvGemmArgs& a);
TileCfg convhalo_pick(int64_t m, int nout, int h, int w, bool bt, bool any_grid = false);
hipError_t convhalo_launch(const ConvGemmArgs& a, const TileCfg& t, hipStream_t s, int cls);
// forward convolution of a narrow input (cs = ci < 8, one phase, wt = OHWI weights with
// K = taps * ci packed densely); rows per tile and columns per tile of narrow_pick
TileCfg narrow_pick(int nout);
hipError_t convnarrow_launch(const ConvGemmArgs& a, const TileCfg& t, hipStream_t s);

// 8-channel repacking of a narrow (ci < 8) NHWC tensor, and extraction of ci channels
// from a weight gradient computed on the repacked layout
hipError_t pack8_launch(const bf16_t* src, int64_t src_pix, int ci, int64_t n, bf16_t* dst, hipStream_t s);
hipError_t unpack_dw_launch(const float* dw8, float* dw, int64_t rows, int ci, int accumulate, hipStream_t s);

// data gradient of a narrow input (ci < 8), one thread per input pixel
struct NarrowDgradArgs {
  const bf16_t* dy;
  int64_t dy_pix;
  const bf16_t* wt;  // OHWI, [co][kh][kw][ci]
  bf16_t* dx;
  int64_t dx_pix;
  int32_t n, h, w, co, kh, kw, sh, sw, ph, pw, ho, wo;
  int32_t accumulate;
};
// wf: workspace for the weights as fp32 [kh][kw][co][ci] (kh * kw * co * ci * 4 bytes)
hipError_t dgrad_narrow_launch(const NarrowDgradArgs& a, int ci, float* wf, hipStream_t s);

// merge per-tile (mean, M2) partials into batch mean / biased variance, fixed order
hipError_t stats_merge_launch(const float2* part, int mtiles, int tile_rows, int64_t m, int c, float* mean_var,
                              hipStream_t s);

// dgrad weight re-layout: for each stride phase, wt[c][tap][o] = w[o][r][s][c] for
// c < ci and 0 for ci <= c < cpad (phase_first counts cpad rows of channels)
struct PhaseTaps {
  int count;
  int r[kMaxTaps], s[kMaxTaps];
};
hipError_t dgrad_weights_launch(const bf16_t* w, bf16_t* wt, int co, int kh, int kw, int ci, int cpad,
                                const int* phase_first, const PhaseTaps* phases, int nphase, hipStream_t s);

// weight gradient: split-K implicit GEMM and its fixed-order reduction
struct WgradArgs {
  const bf16_t* x;
  int64_t x_pix;
  const bf16_t* dy;
  int64_t dy_pix;
  int32_t n, h, w, ci, co, kh, kw, sh, sw, ph, pw, ho, wo;
  int64_t m;            // n * ho * wo
  int32_t ktot;         // kh * kw * ci
  int32_t splits;       // number of reduction ranges
  int64_t rows_per_split;  // multiple of the reduction step
  float* out;           // splits == 1: dw (accumulate honoured); else partials [splits][co][ktot]
  int32_t accumulate;
  int32_t remap;        // set by wgrad_launch: XCD-aware tile order (see xcd_remap)
};
int wgrad_pick_splits(int64_t m, int co, int ktot, int64_t* rows_per_split);
hipError_t wgrad_launch(const WgradArgs& a, hipStream_t s);
hipError_t splitk_reduce_launch(const float* part, int splits, int64_t count, float* dw, int accumulate,
                                hipStream_t s);
// weight gradient of the RGB image layer's shape (3 channels, 3x3, stride 2, padding 1,
// c_out <= 64 and a multiple of 8, output rows a multiple of 4 and columns of 64):
// per-block partials [blocks][c_out][27] in part, then their split reduction into a.out
// (accumulate honoured); x is read with any pixel stride
bool wgrad_stem_shape(const WgradArgs& a);
int wgrad_stem_blocks(const WgradArgs& a);
hipError_t wgrad_stem_launch(const WgradArgs& a, float* part, hipStream_t s);
// weight gradient of a 3x3, stride-1, padding-1 convolution staged by pixel patches (c_in a
// multiple of 32 or 48, c_out of 8, pixel strides of 8, image sides the patch divides), and
// of a 1x1 stride-1 one in steps of 64 pixels (c_in a multiple of 96, 144, 192 or 288):
// wgrad_halo_plan says whether it applies and fills in its split count and patches per
// split; wgrad_halo_launch takes those in a.splits and a.rows_per_split and writes
// partials [splits][c_out][kh kw c_in] to a.out when splits > 1, else dW (accumulate
// honoured)
struct WhGeom {
  int32_t pcols, ppi;   // patches per image row band, per image
  int32_t pps, npatch;  // patches per split, in all
  FastDiv dppi, dpcols;
};
bool wgrad_halo_plan(const WgradArgs& a, int* splits, int64_t* patches_per_split);
hipError_t wgrad_halo_launch(const WgradArgs& a, hipStream_t s);

// BN + SiLU
struct BnArgs {
  int32_t c;
  int64_t m;
  float eps, momentum;
  int64_t y_pix, a_pix, r_pix, dy_pix;
};
int bn_reduce_blocks(int64_t m, int c);
hipError_t bn_stats_launch(const BnArgs& a, const bf16_t* y, float* part3, int nblocks, float* mean_var,
                           hipStream_t s);
// save_mean == nullptr: no saved or running statistics (inference with running statistics)
hipError_t bn_fwd_launch(const BnArgs& a, const bf16_t* y, const float* mean, const float* var, const float* gamma,
                         const float* beta, const bf16_t* res, bf16_t* out, float* save_mean, float* save_rstd,
                         float* run_mean, float* run_var, hipStream_t s);
// coef: workspace for 4 * c folded constants (bn_bwd_fold), written by the finalize;
// dy == nullptr: the reduce and finalize only (dgamma, dbeta), no apply
hipError_t bn_bwd_launch(const BnArgs& a, const bf16_t* g, const bf16_t* y, const float* save_mean,
                         const float* save_rstd, const float* gamma, const float* beta, bf16_t* dy, float* dgamma,
                         float* dbeta, bf16_t* res_grad, float* part2, int nblocks, float* coef, hipStream_t s);

// SPPF max pool (5x5, stride 1, padding 2) and nearest 2x upsampling (pool.hip): n, h, w
// of the pooled / low-resolution tensor, c channels (a multiple of 8), pixel strides of x
// (and dx) and y (and dy); idx: one byte per element of y, dense [n][h][w][c]
struct PoolArgs {
  int32_t n, h, w, c;
  int64_t x_pix, y_pix;
};
hipError_t maxpool5_fwd_launch(const PoolArgs& a, const bf16_t* x, bf16_t* y, uint8_t* idx, hipStream_t s);
hipError_t maxpool5_bwd_launch(const PoolArgs& a, const bf16_t* dy, const uint8_t* idx, bf16_t* dx, int accumulate,
                               hipStream_t s);
hipError_t upsample2x_fwd_launch(const PoolArgs& a, const bf16_t* x, bf16_t* y, hipStream_t s);
hipError_t upsample2x_bwd_launch(const PoolArgs& a, const bf16_t* dy, bf16_t* dx, int accumulate, hipStream_t s);

// Optimiser step (optim.hip): global-norm clip + SGD-Nesterov over a device table of fp32
// tensors.  OptTensor has the layout of numbat_param_tensor.
struct OptTensor {
  float* w;
  const float* g;
  float* mom;
  int64_t n;
  int32_t group;
  int32_t reserved;
};
constexpr int kOptMaxGroups = 8;
constexpr int kOptMaxTensors = 1024;  // the table is staged in LDS (40 bytes each)
constexpr int kOptBlocks = 1024;      // blocks of both launches; part holds kOptBlocks doubles
struct OptGroups {
  int32_t count;
  float lr[kOptMaxGroups], wd[kOptMaxGroups];
};
hipError_t opt_clip_sgd_launch(const OptTensor* tab, int count, const OptGroups& grp, float momentum, float max_norm,
                               float* total_norm, double* part, hipStream_t s);

}  // namespace numbat
