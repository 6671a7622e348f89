// Internal launcher interface between the host orchestration (stage.cpp) and
// the HIP kernels.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"

namespace pulse {

constexpr int MAX_SEG = 3;

// A contiguous range of the implicit operand: K in CONV mode, N in WGRAD
// mode.  It is a 3x3 (taps = 9, zero padded) or 1x1 (taps = 1) conv over the
// virtual input `in` of C channels, so it spans taps * C indices ordered
// (tap, channel) -- the OHWI order of the weights.
struct Seg {
  int begin, end;
  int taps;
  int C;
  VIn in;
  float* grad;  // WGRAD: accumulation target, rows of length end - begin
};

struct GemmArgs {
  Geo g;
  int M, N, K;
  int nseg;
  Seg seg[MAX_SEG];
  // CONV mode
  const void* Bw;      // [N][ldb] weights in the compute dtype
  int ldb;
  const float* bias;   // [N] or null
  const float* rowvec; // [B][N] or null, added to every pixel of image b
  VIn resid;           // residual added in the epilogue (resid.s0.ptr null: none)
  void* out;           // [P][ldo]
  void* out2;          // optional second copy of out
  int out_dtype;
  int ldo;
  int ksplit;          // K splits (conv mode, LDS-DMA path): > 1 writes fp32
  int ksteps;          // partials to part and a finalize applies the epilogue;
                       // ksteps = K-steps per split
  // WGRAD mode
  VIn gy;              // output gradient, M channels
  int kchunk;          // pixels per split
  float* part;         // [splits][M][N] fp32 partials (both modes)
  int wdirect;         // set by the wgrad launcher: one pixel split, so the
                       // epilogue adds its tile into the segment gradients
                       // (one writer per element) and no finalize runs
  // CONV mode of the LDS-DMA kernels without a K split, when H*W % BM == 0:
  // per-channel sum and sum of squares of the output as stored (bf16), one
  // row per (image, M-tile): [B][H*W / BM][2][N]; null: not computed
  float* stats;
  // Same conditions: the GroupNorm+SiLU backward sums of the output taken as
  // the gradient da of a = SiLU(GN(x)): per channel, sum dz and sum dz*xhat
  // with dz = da (as stored) * SiLU'(x*scale + shift) and xhat =
  // (x - mean) * rstd, one row per (image, M-tile): [B][H*W / BM][2][N];
  // null: not computed.  scale/shift [B][N], mean/rstd [B][gnb_G].
  float* gnb;
  VIn gnb_x;
  const float* gnb_scale;
  const float* gnb_shift;
  const float* gnb_mean;
  const float* gnb_rstd;
  int gnb_G;
  // host side, K split: launch only the GEMM (the caller runs
  // launch_splitk_finalize_stats, which also reduces the statistics)
  int skip_finalize;
  // set by the launchers of igemm2.hip (callers leave them 0): multiply-high
  // reciprocals of the kernels' runtime divisors, each exact over the range
  // it divides, or 0 where the kernel divides (see rcp_u32)
  uint32_t rcp_w, rcp_h, rcp_hw, rcp_nt, rcp_tn;
  uint32_t rcp_segc[3];
};

// Multiply-high reciprocal of d for quotients n / d with n <= nmax:
// M = floor((2^32 - 1) / d) + 1 gives floor(n / d) = mulhi(n, M) whenever
// n < 2^32 / d (the rounding error n (M - 2^32 / d) / 2^32 stays below
// 1 / d).  0 where d < 2 or the range is too wide.
inline uint32_t rcp_u32(uint64_t d, uint64_t nmax) {
  if (d < 2 || nmax >= (1ull << 32) / d) return 0;
  return (uint32_t)(0xffffffffull / d + 1);
}

// implicit GEMM, register-staged (igemm.hip): the fp32 stage and bf16
// channel counts that are multiples of 32 but not of 64
enum Tile : int {
  TILE_128x128_K32 = 0,  // bf16, 32 channels per K-step
  TILE_64x64_F32 = 1,    // fp32, 32 channels per K-step
  TILE_COUNT = 2
};
struct TileInfo {
  int bm, bn, bk;
  int per_cu;  // blocks resident per CU (LDS-limited), 0 when not known
};
TileInfo tile_info(int tile);
hipError_t launch_conv(const GemmArgs& a, int tile, hipStream_t st);
hipError_t launch_wgrad(const GemmArgs& a, int tile, int splits, hipStream_t st);
hipError_t launch_wgrad_finalize(const GemmArgs& a, int splits, hipStream_t st);

// second generation (igemm2.hip): LDS-DMA operand loads, bf16 with 64
// channels per K-step.  zero16: 16 zero bytes of device memory.
enum Tile2 : int {
  TILE2_C128x160 = 0,   // 4 waves of 64 x 80, two blocks per CU
  TILE2_C128x128 = 1,   // 4 waves of 64 x 64, two blocks per CU
  TILE2_C128x192 = 2,   // 4 waves of 64 x 96, two blocks per CU
  TILE2_C64x128S3 = 3,  // 4 waves of 32 x 64, three LDS stages, two blocks per CU
  TILE2_CONV_LAST = 3,
  TILE2_W320x128 = 20,  // 8 waves of 80 x 64, one block per CU
  TILE2_W128x128 = 21,  // 4 waves of 64 x 64
  TILE2_WGRAD_FIRST = 20,
  TILE2_WGRAD_LAST = 21
};
TileInfo tile2_info(int tile);
// t0 / t1 (may be null): events recorded by the GEMM kernel's own start and
// by the completion of the launch's last kernel (the GEMM or its K-split
// finalize), which time the launch without marker packets around it.
hipError_t launch_conv2(const GemmArgs& a, int tile, hipStream_t st, hipEvent_t t0 = nullptr,
                        hipEvent_t t1 = nullptr);
hipError_t launch_wgrad2(const GemmArgs& a, int tile, int splits, const void* zero16,
                         hipStream_t st);

// ---- GroupNorm / reductions (norm.hip) -----------------------------------

// Grid shape shared by the per-channel reduction kernels: image b, pixel
// chunk of `cp` pixels, a block of vx channel vectors x py pixel lanes, zb
// blocks across the channel vectors.
struct RedGrid {
  int chunks, cp;
  int vx, py, zb;
};
RedGrid red_grid(const Geo& g, int C);

// partial[b][chunk][2][C]: per-channel sum and sum of squares of x.
// copy (null: none): the channels below x.c0 of x as read, [P][x.c0]
hipError_t launch_gn_stats_partial(const VIn& x, const Geo& g, RedGrid rg, float* partial,
                                   hipStream_t st, void* copy = nullptr);
// mean/rstd [B][G] and the folded affine scale/shift [B][C].
// K-split conv finalize that also reduces the output: out = sum_z part[z]
// (fixed order) + bias + rowvec + residual (bf16), and the per-channel sum
// and sum of squares of the stored output per (image, chunk of the reduction
// grid rg over N channels) row of a.stats.
hipError_t launch_splitk_finalize_stats(const GemmArgs& a, RedGrid rg, hipStream_t st,
                                        hipEvent_t done = nullptr);
hipError_t launch_gn_stats_finalize(const float* partial, const Geo& g, RedGrid rg, int C,
                                    int G, float eps, const float* gamma, const float* beta,
                                    float* mean, float* rstd, float* scale, float* shift,
                                    hipStream_t st);
// a = SiLU(x * scale + shift); channels < x.c0 go to dst0, the rest to dst1.
hipError_t launch_gn_apply(const VIn& x, const Geo& g, const float* scale,
                           const float* shift, void* dst0, void* dst1, int dtype,
                           hipStream_t st);

// GroupNorm+SiLU backward.  da: gradient w.r.t. SiLU(GN(x)) ([P][C], any dtype).
// partial[b][chunk][0][c] = sum dz, [1][c] = sum dz * xhat with
// dz = da * SiLU'(z), z = x * scale + shift, xhat = (x - mean) * rstd.
hipError_t launch_gn_bwd_partial(const Src& da, const VIn& x, const Geo& g, RedGrid rg,
                                 const float* scale, const float* shift, const float* mean,
                                 const float* rstd, int G, float* partial, hipStream_t st);
// coef[b][g][2] = (sum_g gamma*dz, sum_g gamma*dz*xhat) / count, and
// dgamma[c] += sum dz*xhat, dbeta[c] += sum dz.
hipError_t launch_gn_bwd_finalize(const float* partial, const Geo& g, RedGrid rg, int C,
                                  int G, const float* gamma, float* coef, float* dgamma,
                                  float* dbeta, hipStream_t st);

struct GnBwdOut {
  void* dst0;      // channels [0, c_split): stride c_split
  int dtype0;
  void* dst1;      // channels [c_split, C): stride C - c_split (may be null if c_split == C)
  int dtype1;
  int c_split;
  VIn add0;        // optional addend (add0.s0.ptr null: none), C channels
  const float* add1;  // optional fp32 addend [P][C]
  float* chan_partial;  // optional per-(b, chunk, c) sums of the output
};
// dx = rstd * (gamma*dz - coef0 - xhat*coef1) + addends, split-stored.
// done (may be null): an event recorded by the kernel's own completion.
hipError_t launch_gn_bwd_apply(const Src& da, const VIn& x, const Geo& g, RedGrid rg,
                               const float* scale, const float* shift, const float* mean,
                               const float* rstd, const float* gamma, const float* coef,
                               int G, const GnBwdOut& o, hipStream_t st,
                               hipEvent_t done = nullptr);

// partial[b][chunk][0][c] = sum over the chunk of v (v may carry an addend).
hipError_t launch_chan_sum_partial(const VIn& v, const Geo& g, RedGrid rg, float* partial,
                                   hipStream_t st);
// pi[s][b][c] = sum_chunk partial[b][chunk][s][c] for s < nslot (pi: [nslot][B][C]).
hipError_t launch_chan_per_image(const float* partial, const Geo& g, RedGrid rg, int C,
                                 int nslot, float* pi, hipStream_t st);
// acc0 (and dup) += sum of slot 0, acc1 += sum of slot 1 over every image and
// chunk, in one pass (no per-image sums)
hipError_t launch_chan_totals(const float* partial, const Geo& g, RedGrid rg, int C, int nslot,
                              float* acc0, float* dup, float* acc1, hipStream_t st);

// ---- timestep embedding, weights, copies (misc.hip) ----------------------

// e[b][o] = bias_a[o] + bias_b[o] + sum_d Wl[o][d] * SiLU(temb[b][d])
hipError_t launch_temb_fwd(const void* temb, int dtype, int B, int D, int O, const float* Wl,
                           const float* bias_a, const float* bias_b, float* e,
                           hipStream_t st);
// The projections of several stage blocks from one temb in one launch:
// blk[k].e[b][o] (row stride ldE) for every block k < n; copy (null: none)
// receives temb itself.
constexpr int TEMB_MAX_BLOCKS = 16;
struct TembFwdBlock {
  const float* Wl;      // [O][D]
  const float* bias_a;  // [O]
  const float* bias_b;  // [O] or null
  float* e;             // [B][ldE]
  int O, ldE;
};
struct TembFwdSet {
  TembFwdBlock blk[TEMB_MAX_BLOCKS];
  int n;
};
hipError_t launch_temb_fwd_multi(const void* temb, int dtype, int B, int D,
                                 const TembFwdSet& set, void* copy, hipStream_t st);
// dWl += de^T SiLU(temb); dbl += sum_b de; db1 += sum_b de;
// dtemb += (de Wl) * SiLU'(temb) (dtemb may be null).
hipError_t launch_temb_bwd(const float* de, const void* temb, int dtype, int B, int D, int O,
                           const float* Wl, float* dWl, float* dbl, float* db1, float* dtemb,
                           hipStream_t st);

// dst[r][col_off + c] = (dtype) src[r][c] for r < rows, c < cols.
hipError_t launch_convert_rows(const float* src, int rows, int cols, void* dst, int ldd,
                               int col_off, int dtype, hipStream_t st);
// 3x3 data-gradient weights: dst[c][8 - tap][o] = src[o][tap][c].
hipError_t launch_flip3x3(const float* src, int O, int C, void* dst, int dtype,
                          hipStream_t st);
// dst[c][o] = src[o][c]
hipError_t launch_transpose(const float* src, int O, int C, void* dst, int dtype,
                            hipStream_t st);
// dst[i] = a[i] + (b ? b[i] : 0)
hipError_t launch_vec_add(const float* a, const float* b, float* dst, int n, hipStream_t st);
// dst = (ddt)(a + b) elementwise, a of dtype adt, b fp32
hipError_t launch_add_cast(const void* a, int adt, const float* b, void* dst, int ddt, long n,
                           hipStream_t st);
// dst = convert(src), n elements (dtypes as DType)
hipError_t launch_cast(const void* src, int sdt, void* dst, int ddt, long n, hipStream_t st);

}  // namespace pulse
