// Host side of the transformer-block stage: descriptor validation, parameter
// and workspace layout, per-microbatch bookkeeping and the kernel sequence of
// every forward / backward half.  Implements include/pulse_tstage.h.
//
// Every linear layer runs on the implicit-GEMM kernels (igemm2.hip) in their
// 1x1 form over a [batch, 1, tokens] geometry: the forward and the data
// gradient in conv mode (out[T][N] = in[T][K] W^T with W given as [N][K]),
// the weight gradient in wgrad mode.  The decoder's skip linear reads
// [v || skip] as one two-source operand, so the concatenation never exists
// in memory (Sec. III), and its data gradient is produced as two GEMMs over
// the two row halves of the transposed weight: the upstream part (dL/dv)
// and the skip part, which is buffered in fp32 in the microbatch's row until
// the encoder's backward adds it (Sec. I).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "error.hpp"
#include "kernels.hpp"
#include "pulse_tstage.h"
#include "tkernels.hpp"

using namespace pulse;

namespace {

pulse_status tfail(pulse_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  return set_last_error(s, buf);
}

#define THIP(expr)                                                                     \
  do {                                                                                 \
    hipError_t e_ = (expr);                                                            \
    if (e_ != hipSuccess)                                                              \
      return tfail(PULSE_E_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));        \
  } while (0)

#define TCHK(expr)                                                                     \
  do {                                                                                 \
    pulse_status s_ = (expr);                                                          \
    if (s_ != PULSE_OK) return s_;                                                     \
  } while (0)

size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

struct TParam {
  std::string name;
  int64_t off;
  int32_t shape[4];
};

// One transformer block: parameter offsets, bf16 weight copies (workspace
// offsets; w_* [out][in], t_* [in][out]) and the row offsets of what its
// backward reads.
struct TBlock {
  bool dec = false;
  int64_t ln1g, ln1b, qkvW, qkvb, projW, projb, ln2g, ln2b, fc1W, fc1b, fc2W, fc2b;
  int64_t skW = -1, skb = -1;
  size_t w_qkv, w_proj, w_fc1, w_fc2, t_qkv, t_proj, t_fc1, t_fc2, w_sk = 0, t_sk = 0;
  size_t r_x = 0;  // block input kept in the row (encoder block 0: the stage input;
                   // decoder block: the skip linear's output)
  size_t r_v = 0;  // decoder: upstream input v of the skip linear
  size_t r_a, r_st1, r_qkv, r_lse, r_o, r_h, r_a2, r_st2, r_z, r_m;
};

enum TRowState { T_FREE = 0, T_ENC_FWD = 1, T_DEC_FWD = 2, T_DEC_BWD = 3 };

struct TRow {
  int mb = -1;
  int state = T_FREE;
};

struct TTimed {
  hipEvent_t a, b;
  double flops, bytes;
};

}  // namespace

// Scratch buffers of one parity that the side stream may still read, with
// the event that frees each (null: free).
struct SideReads {
  hipEvent_t dy = nullptr, dm = nullptr, dh = nullptr, dqkv = nullptr, dsx = nullptr;
};

struct pulse_tstage {
  pulse_tstage_desc d{};
  bool dry = false;
  int B = 0, L = 0, C = 0, H = 0, R = 0;  // R: MLP hidden width
  long T = 0;
  Geo geo{};
  std::vector<TParam> params;
  int64_t n_params = 0;
  std::vector<TBlock> eb, db;
  // workspace
  size_t ws_bytes = 0, off_rows = 0, row_size = 0;
  size_t row_slot[64] = {}, row_sgrad[64] = {};
  // gradients that the side stream reads come in two copies, one per block
  // parity, so that a block overwrites only what the block before the
  // previous one left (the side stream rarely lags that far)
  size_t s_dy[2] = {0, 0}, s_dm[2] = {0, 0}, s_da2 = 0, s_dh[2] = {0, 0}, s_do = 0,
         s_dqkv[2] = {0, 0}, s_da = 0, s_dsx[2] = {0, 0}, s_dv = 0, s_dsum = 0, s_kpart = 0,
         s_wpart = 0, s_red = 0, s_zero = 0;
  size_t kpart_cap = 0, wpart_cap = 0, red_cap = 0;
  size_t s_red2 = 0;  // reduction buffer of the side stream
  // column-sum partials of dh (LN2 backward) and of a decoder block's
  // skip-linear output gradient (LN1 backward): the bias gradients of proj
  // and skip without another pass over them
  size_t s_cs_h[2] = {0, 0}, s_cs_x[2] = {0, 0};
  // side stream: the weight-gradient GEMMs and bias-gradient sums of the
  // backward pass run on it, concurrently with the data-gradient chain
  hipStream_t side = nullptr;
  std::vector<hipEvent_t> sev;  // synchronisation events, reused per call
  size_t sev_used = 0;
  // overlapped decoder backward (pulse_tstage_overlap_bwd): a decoder
  // backward may return with its last parameter-gradient work still on the
  // side stream; the next call joins it, except an encoder backward of the
  // same microbatch on the same stream, which continues beside it with the
  // decoder call's side-read events (their pool is not recycled until then)
  bool overlap_bwd = false, join_pending = false;
  int32_t pending_mb = -1;
  hipStream_t pending_st = nullptr;
  SideReads pending_rds[2];
  hipEvent_t pending_dy = nullptr;  // the decoder's last read of a dy buffer
  hipEvent_t ev_settle = nullptr;
  // GEMM tuning overrides (env, read at create; -1: the default choice)
  int conv_tile_force = -1, conv_ks_cap = 16, wgrad_tile_force = -1;
  // binding
  const float* prm = nullptr;
  float* grd = nullptr;
  char* ws = nullptr;
  bool bound = false, synced = false;
  std::vector<TRow> rows;
  // timing
  bool timing = false;
  std::vector<TTimed> timed;
  std::vector<hipEvent_t> ev_pool;
  size_t ev_used = 0;

  char* at(size_t off) const { return ws + off; }
  char* row(int r) const { return ws + off_rows + (size_t)r * row_size; }
  const float* pp(int64_t off) const { return prm + off; }
  float* gp(int64_t off) const { return grd + off; }
  float* fat(size_t off) const { return reinterpret_cast<float*>(ws + off); }
};

namespace {

// ---------------------------------------------------------------------------
// layout
// ---------------------------------------------------------------------------

int64_t add_param(pulse_tstage* s, const std::string& name, int d0, int d1 = 0) {
  TParam p;
  p.name = name;
  p.off = s->n_params;
  p.shape[0] = d0;
  p.shape[1] = d1;
  p.shape[2] = p.shape[3] = 0;
  s->params.push_back(p);
  s->n_params += (int64_t)d0 * (d1 > 0 ? d1 : 1);
  // keep every tensor 16-byte aligned for the vector loads
  s->n_params = (s->n_params + 3) & ~(int64_t)3;
  return p.off;
}

void layout_block_params(pulse_tstage* s, TBlock& b, const std::string& pre) {
  const int C = s->C, R = s->R;
  b.ln1g = add_param(s, pre + "ln1.g", C);
  b.ln1b = add_param(s, pre + "ln1.b", C);
  b.qkvW = add_param(s, pre + "qkv.W", 3 * C, C);
  b.qkvb = add_param(s, pre + "qkv.b", 3 * C);
  b.projW = add_param(s, pre + "proj.W", C, C);
  b.projb = add_param(s, pre + "proj.b", C);
  b.ln2g = add_param(s, pre + "ln2.g", C);
  b.ln2b = add_param(s, pre + "ln2.b", C);
  b.fc1W = add_param(s, pre + "fc1.W", R, C);
  b.fc1b = add_param(s, pre + "fc1.b", R);
  b.fc2W = add_param(s, pre + "fc2.W", C, R);
  b.fc2b = add_param(s, pre + "fc2.b", C);
}

int env_or(const char* name, int dflt) {
  const char* v = getenv(name);
  return (v && *v) ? atoi(v) : dflt;
}

// Tile and K split of a conv-mode GEMM (M x N over K).  Token-major GEMMs
// are short (K of one to four widths), so per-block set-up and the last,
// partly filled round of blocks weigh as much as the MFMA work, and a K
// split costs an fp32 partial of M x N per split.  Default, from sweeps of
// every tile and split on the 768-wide stage: the largest 128-row tile whose
// tile count still fits one round of two blocks per CU (at least 400 tiles
// of 128 x 192, 128 x 160 or 128 x 128), without a K split; a GEMM that
// needs more than one round of 128-row tiles takes 128 x 192 (from the
// sweep of the 1024-token, 1408-wide stage: +13 % step against 64 x 128);
// otherwise 64 x 128 tiles with a three-stage LDS ring (two blocks per CU),
// no K split: with 16 MFMAs per wave and K-step the deeper ring hides the
// operand latency that two stages leave exposed, and beats splitting K.
// Overrides (for sweeps): PULSE_TCONV_TILE forces a tile (with the split
// rule of two blocks per CU, at least 4 K-steps per split),
// PULSE_TCONV_KSPLIT_MAX caps the split.
struct ConvPlan {
  int tile, ks, ksteps;
};

long tile_count(int tile, long M, int N) {
  const TileInfo ti = tile2_info(tile);
  return ((M + ti.bm - 1) / ti.bm) * ((N + ti.bn - 1) / ti.bn);
}

ConvPlan tconv_plan(int tile_force, int ks_cap, long M, int N, int K) {
  ConvPlan p;
  long ks = 1;
  if (tile_force >= 0) {
    p.tile = tile_force;
    const long tiles = tile_count(p.tile, M, N);
    const long kt = K / tile2_info(p.tile).bk;
    if (tiles < 512) {
      ks = (512 + tiles - 1) / tiles;
      ks = std::min(ks, std::max(1L, kt / 4));
    }
  } else {
    p.tile = -1;
    long best = 0;
    for (int t : {TILE2_C128x192, TILE2_C128x160, TILE2_C128x128}) {
      const long n = tile_count(t, M, N);
      if (n <= 512 && n >= 400 && n > best) {
        best = n;
        p.tile = t;
      }
    }
    if (p.tile < 0) p.tile = tile_count(TILE2_C128x192, M, N) > 512 ? TILE2_C128x192 : TILE2_C64x128S3;
  }
  ks = std::min(ks, (long)std::max(1, ks_cap));
  const long kt = K / tile2_info(p.tile).bk;
  p.ksteps = (int)((kt + ks - 1) / ks);
  p.ks = (int)((kt + p.ksteps - 1) / p.ksteps);  // no empty split
  return p;
}

// weight-gradient tile for M rows summed over P tokens (PULSE_TWGRAD_TILE
// forces one).  The 320 x 128 tile (8 waves, one block per CU) does the
// most MFMA work per operand byte but quantises M in steps of 320; it wins
// when M is a multiple of 320, or when every block's token loop is long
// (P >= 8192: measured on the 1024-token, 1408-wide stage, where it cut the
// step by 7 %; at 4096 tokens of the 768-wide stage 128 x 128 is 2 % faster).
int twgrad_tile(int tile_force, int M, long P) {
  if (tile_force >= TILE2_WGRAD_FIRST && tile_force <= TILE2_WGRAD_LAST) return tile_force;
  return M % 320 == 0 || P >= 8192 ? TILE2_W320x128 : TILE2_W128x128;
}

// Token splits of a weight-gradient GEMM (M x N over P tokens): the count
// that minimises rounds(s) * T_tile / s + bytes(s) * M * N / HBM, as for
// the ResBlock stage (bytes(s) = 8 s + 8 for s partials and the finalize,
// 8 for one split added into the gradient in the GEMM epilogue); kchunk
// receives the tokens per split
int twgrad_splits(int tile, long P, int M, int N, int& kchunk) {
  const TileInfo ti = tile2_info(tile);
  const long tiles = (long)((M + ti.bm - 1) / ti.bm) * ((N + ti.bn - 1) / ti.bn);
  const long per_cu = ti.per_cu > 0 ? std::min(ti.per_cu, 2) : 1;
  const long slots = 256L * per_cu;
  const double t_tile = 2.0 * ti.bm * ti.bn * (double)P / 3.0e12;
  const double t_elem = (double)M * N / 4.0e12;
  const long maxs = std::max(1L, P / (4L * ti.bk));
  long best = 1;
  double best_t = 1e30;
  for (long sp = 1; sp <= std::min(maxs, 256L); ++sp) {
    const long rounds = (tiles * sp + slots - 1) / slots;
    const double bytes = sp == 1 ? 8.0 : 8.0 * sp + 8.0;
    const double t = rounds * t_tile / sp + bytes * t_elem;
    if (t < best_t * 0.999) {
      best_t = t;
      best = sp;
    }
  }
  long kc = (P + best - 1) / best;
  kc = (kc + ti.bk - 1) / ti.bk * ti.bk;
  kchunk = (int)kc;
  return (int)((P + kc - 1) / kc);
}

pulse_status tvalidate(const pulse_tstage_desc* d) {
  if (!d) return tfail(PULSE_E_INVALID_ARG, "desc is NULL");
  if (d->dtype != PULSE_BF16) return tfail(PULSE_E_SHAPE, "the transformer stage runs bf16 only");
  if (d->batch < 1) return tfail(PULSE_E_SHAPE, "batch must be >= 1");
  if (d->tokens < 64 || d->tokens > ATTN_LMAX || d->tokens % 64)
    return tfail(PULSE_E_SHAPE, "tokens must be a multiple of 64 in [64, %d]", ATTN_LMAX);
  if (d->heads < 1 || d->width != 64 * d->heads || d->width > 2048)
    return tfail(PULSE_E_SHAPE, "width must be 64 * heads and at most 2048");
  if (d->mlp_ratio < 1 || d->mlp_ratio > 8) return tfail(PULSE_E_SHAPE, "mlp_ratio must be in [1, 8]");
  if (!(d->eps >= 0.0f)) return tfail(PULSE_E_SHAPE, "eps must be >= 0");
  if (d->n_enc < 1 || d->n_enc > 32 || d->n_dec != d->n_enc)
    return tfail(PULSE_E_SHAPE, "n_enc must be in [1, 32] and n_dec == n_enc");
  if (d->max_inflight < 1 || d->max_inflight > 64)
    return tfail(PULSE_E_SHAPE, "max_inflight must be in [1, 64]");
  if ((long)d->batch * d->tokens > (1L << 20)) return tfail(PULSE_E_SHAPE, "too many tokens");
  // the GEMM kernels address each operand through a 32-bit buffer range
  const long widest = std::max(3L * d->width, (long)d->mlp_ratio * d->width);
  if ((long)d->batch * d->tokens * widest * 2 >= (1L << 31))
    return tfail(PULSE_E_SHAPE, "an activation of batch * tokens * max(3 width, mlp width) "
                                "bf16 values must stay below 2 GiB");
  return PULSE_OK;
}

void build_layout(pulse_tstage* s) {
  const int C = s->C, R = s->R, ne = s->d.n_enc, nd = s->d.n_dec;
  const long T = s->T;
  s->eb.resize(ne);
  s->db.resize(nd);
  for (int k = 0; k < ne; ++k) layout_block_params(s, s->eb[k], "enc" + std::to_string(k) + ".");
  for (int k = 0; k < nd; ++k) {
    TBlock& b = s->db[k];
    b.dec = true;
    const std::string pre = "dec" + std::to_string(k) + ".";
    b.skW = add_param(s, pre + "skip.W", C, 2 * C);
    b.skb = add_param(s, pre + "skip.b", C);
    layout_block_params(s, b, pre);
  }
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += al256(bytes);
    return o;
  };
  // bf16 weight copies
  const size_t wq = (size_t)3 * C * C * 2, wp = (size_t)C * C * 2, wf = (size_t)R * C * 2;
  for (auto* v : {&s->eb, &s->db})
    for (TBlock& b : *v) {
      b.w_qkv = take(wq);
      b.t_qkv = take(wq);
      b.w_proj = take(wp);
      b.t_proj = take(wp);
      b.w_fc1 = take(wf);
      b.t_fc1 = take(wf);
      b.w_fc2 = take(wf);
      b.t_fc2 = take(wf);
      if (b.dec) {
        b.w_sk = take(2 * wp);
        b.t_sk = take(2 * wp);
      }
    }
  // shared scratch of the backward pass
  const size_t act = (size_t)T * C * 2;
  const size_t lbytes = (size_t)s->B * s->H * s->L * 4;  // one fp32 per (image, head, token)
  s->s_dy[0] = take(act);
  s->s_dy[1] = take(act);
  for (int i = 0; i < 2; ++i) {
    s->s_dm[i] = take((size_t)T * R * 2);
    s->s_dh[i] = take(act);
    s->s_dqkv[i] = take(3 * act);
    s->s_dsx[i] = take(act);
  }
  s->s_da2 = take(act);
  s->s_do = take(act);
  s->s_da = take(act);
  s->s_dv = take(act);
  s->s_dsum = take(lbytes);
  // partial buffers: the largest conv K split and weight-gradient split
  size_t kcap = 0, wcap = 0;
  const int gemms[][3] = {{3 * C, C, 0}, {C, C, 0}, {R, C, 0}, {C, R, 0}, {C, 2 * C, 0},
                          {C, 3 * C, 0}, {C, R, 0}, {R, C, 0}};
  for (const auto& g : gemms) {
    // as a conv: N = g[0] columns over K = g[1]; as a weight gradient: M = g[0]
    const int N = g[0], K = g[1];
    const ConvPlan cp = tconv_plan(s->conv_tile_force, s->conv_ks_cap, T, N, K);
    if (cp.ks > 1) kcap = std::max(kcap, (size_t)cp.ks * T * N);
    int kc = 0;
    const int sp = twgrad_splits(twgrad_tile(s->wgrad_tile_force, N, T), T, N, K, kc);
    wcap = std::max(wcap, (size_t)sp * N * K);
  }
  s->kpart_cap = kcap;
  s->wpart_cap = wcap;
  s->s_kpart = take(std::max<size_t>(kcap, 4) * 4);
  s->s_wpart = take(std::max<size_t>(wcap, 4) * 4);
  // reductions: LayerNorm partials [blocks][2][C] and bias-gradient chunk
  // partials [chunks <= 128][2][N <= max(3C, R)]
  const size_t red = std::max((size_t)ln_bwd_blocks(T) * 2 * C,
                              (size_t)128 * 2 * std::max(3 * C, R));
  s->red_cap = red;
  s->s_red = take(red * 4);
  s->s_red2 = take(red * 4);
  for (int i = 0; i < 2; ++i) {
    s->s_cs_h[i] = take((size_t)ln_bwd_blocks(T) * 2 * C * 4);
    s->s_cs_x[i] = take((size_t)ln_bwd_blocks(T) * 2 * C * 4);
  }
  s->s_zero = take(256);
  // per-microbatch rows
  s->off_rows = off;
  size_t ro = 0;
  auto rtake = [&](size_t bytes) {
    const size_t o = ro;
    ro += al256(bytes);
    return o;
  };
  const size_t stb = (size_t)T * 8;
  auto block_rows = [&](TBlock& b) {
    b.r_a = rtake(act);
    b.r_st1 = rtake(stb);
    b.r_qkv = rtake(3 * act);
    b.r_lse = rtake(lbytes);
    b.r_o = rtake(act);
    b.r_h = rtake(act);
    b.r_a2 = rtake(act);
    b.r_st2 = rtake(stb);
    b.r_z = rtake((size_t)T * R * 2);
    b.r_m = rtake((size_t)T * R * 2);
  };
  s->eb[0].r_x = rtake(act);
  for (TBlock& b : s->eb) block_rows(b);
  for (int k = 0; k < ne; ++k) {
    s->row_slot[k] = rtake(act);
    s->row_sgrad[k] = rtake((size_t)T * C * 4);
  }
  for (TBlock& b : s->db) {
    b.r_v = rtake(act);
    b.r_x = rtake(act);
    block_rows(b);
  }
  s->row_size = al256(ro);
  s->ws_bytes = off + s->row_size * s->d.max_inflight;
}

// ---------------------------------------------------------------------------
// GEMM and reduction helpers
// ---------------------------------------------------------------------------

VIn tvin(const void* p, int C) {
  VIn v;
  v.s0 = Src{p, DT_BF16, C};
  v.s1 = Src{nullptr, DT_BF16, 0};
  v.c0 = C;
  v.C = C;
  v.add = nullptr;
  return v;
}

VIn tvin2(const void* p0, int c0, const void* p1, int c1) {
  VIn v;
  v.s0 = Src{p0, DT_BF16, c0};
  v.s1 = Src{p1, DT_BF16, c1};
  v.c0 = c0;
  v.C = c0 + c1;
  v.add = nullptr;
  return v;
}

VIn tnone() {
  VIn v{};
  v.s0.ptr = nullptr;
  return v;
}

Seg tseg(int K, const VIn& in, float* grad = nullptr) {
  Seg g;
  g.begin = 0;
  g.end = K;
  g.taps = 1;
  g.C = K;
  g.in = in;
  g.grad = grad;
  return g;
}

GemmArgs tbase(const pulse_tstage* s) {
  GemmArgs a;
  std::memset(&a, 0, sizeof a);
  a.g = s->geo;
  a.resid = tnone();
  a.gy = tnone();
  return a;
}

hipEvent_t next_event(pulse_tstage* s) {
  if (s->ev_used == s->ev_pool.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    s->ev_pool.push_back(e);
  }
  return s->ev_pool[s->ev_used++];
}

// out[T][N] = in[T][K] W^T (+ bias) (+ resid), W bf16 [N][ldb]; out2 an
// optional second copy; out_dtype DT_BF16 or DT_F32
pulse_status linear(pulse_tstage* s, int N, const Seg& in, const void* W, int ldb,
                    const float* bias, const void* resid, void* out, void* out2, int out_dtype,
                    hipStream_t st) {
  GemmArgs a = tbase(s);
  a.M = (int)s->T;
  a.N = N;
  a.K = in.end;
  a.nseg = 1;
  a.seg[0] = in;
  a.Bw = W;
  a.ldb = ldb;
  a.bias = bias;
  if (resid) a.resid = tvin(resid, N);
  a.out = out;
  a.out2 = out2;
  a.out_dtype = out_dtype;
  a.ldo = N;
  const ConvPlan cp = tconv_plan(s->conv_tile_force, s->conv_ks_cap, s->T, N, a.K);
  const int tile = cp.tile;
  a.ksplit = cp.ks;
  a.ksteps = cp.ksteps;
  if (cp.ks > 1) {
    if ((size_t)cp.ks * a.M * N > s->kpart_cap)
      return tfail(PULSE_E_SHAPE, "internal: conv partial buffer too small");
    a.part = s->fat(s->s_kpart);
  }
  // timed launches: the kernels record the events at their start and completion
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (s->timing) {
    e0 = next_event(s);
    e1 = next_event(s);
  }
  const bool timed = e0 && e1;
  THIP(launch_conv2(a, tile, st, timed ? e0 : nullptr, timed ? e1 : nullptr));
  if (timed) {
    const double P = (double)a.M;
    const double bytes = P * a.K * 2.0 + (double)N * a.K * 2.0 + (resid ? P * N * 2.0 : 0.0) +
                         P * N * (out_dtype == DT_BF16 ? 2.0 : 4.0) * (out2 ? 2.0 : 1.0);
    s->timed.push_back(TTimed{e0, e1, 2.0 * P * N * a.K, bytes});
  }
  return PULSE_OK;
}

// grad[M][in.end] += gy[T][M]^T in[T][K]
pulse_status linear_wgrad(pulse_tstage* s, int M, const Seg& in, const void* gy,
                          hipStream_t st) {
  GemmArgs a = tbase(s);
  a.M = M;
  a.N = in.end;
  a.K = (int)s->T;
  a.nseg = 1;
  a.seg[0] = in;
  a.gy = tvin(gy, M);
  int kc = 0;
  const int wtile = twgrad_tile(s->wgrad_tile_force, M, s->T);
  const int splits = twgrad_splits(wtile, s->T, M, a.N, kc);
  if ((size_t)splits * M * a.N > s->wpart_cap)
    return tfail(PULSE_E_SHAPE, "internal: weight-gradient partial buffer too small");
  a.kchunk = kc;
  a.part = s->fat(s->s_wpart);
  THIP(launch_wgrad2(a, wtile, splits, s->at(s->s_zero), st));
  return PULSE_OK;
}

// acc[n] += sum over the T tokens of v[t][n] (part: a reduction buffer)
pulse_status col_sum(pulse_tstage* s, const void* v, int N, float* acc, float* part,
                     hipStream_t st) {
  const Geo g{1, (int)s->T, 1};
  const RedGrid rg = red_grid(g, N);
  if ((size_t)rg.chunks * 2 * N > s->red_cap)
    return tfail(PULSE_E_SHAPE, "internal: reduction buffer too small");
  THIP(launch_chan_sum_partial(tvin(v, N), g, rg, part, st));
  THIP(launch_chan_totals(part, g, rg, N, 1, acc, nullptr, nullptr, st));
  return PULSE_OK;
}

// acc[n] += sum of rows [0, rows) of partials laid out [rows][2][N] (row 0)
pulse_status totals(const float* part, int rows, int N, float* acc, hipStream_t st) {
  RedGrid rg{};
  rg.chunks = rows;
  THIP(launch_chan_totals(part, Geo{1, 1, 1}, rg, N, 1, acc, nullptr, nullptr, st));
  return PULSE_OK;
}

// LayerNorm backward: dx = add + dLN(dy); g/b gradients accumulated; csum
// (or null) receives the column-sum partials of dx
pulse_status ln_backward(pulse_tstage* s, const void* dy, const void* x, const float* stats,
                         int64_t goff, int64_t boff, const void* add, void* dx,
                         hipStream_t st, float* csum = nullptr) {
  const int nb = ln_bwd_blocks(s->T);
  float* part = s->fat(s->s_red);
  THIP(launch_ln_bwd(dy, x, stats, s->pp(goff), add, s->T, s->C, dx, part, csum, st));
  RedGrid rg{};
  rg.chunks = nb;
  THIP(launch_chan_totals(part, Geo{1, 1, 1}, rg, s->C, 2, s->gp(goff), nullptr, s->gp(boff),
                          st));
  return PULSE_OK;
}

// ---------------------------------------------------------------------------
// block forward / backward
// ---------------------------------------------------------------------------

pulse_status block_fwd(pulse_tstage* s, char* row, const TBlock& b, const void* x, void* out,
                       void* out2, hipStream_t st) {
  const int C = s->C, R = s->R;
  const float eps = s->d.eps;
  void* a = row + b.r_a;
  float* st1 = reinterpret_cast<float*>(row + b.r_st1);
  void* qkv = row + b.r_qkv;
  void* o = row + b.r_o;
  void* h = row + b.r_h;
  void* a2 = row + b.r_a2;
  float* st2 = reinterpret_cast<float*>(row + b.r_st2);
  void* z = row + b.r_z;
  void* m = row + b.r_m;
  THIP(launch_ln_fwd(x, s->T, C, eps, s->pp(b.ln1g), s->pp(b.ln1b), a, st1, st));
  TCHK(linear(s, 3 * C, tseg(C, tvin(a, C)), s->at(b.w_qkv), C, s->pp(b.qkvb), nullptr, qkv,
              nullptr, DT_BF16, st));
  THIP(launch_attn_fwd(qkv, s->B, s->L, C, s->H, o, reinterpret_cast<float*>(row + b.r_lse), st));
  TCHK(linear(s, C, tseg(C, tvin(o, C)), s->at(b.w_proj), C, s->pp(b.projb), x, h, nullptr,
              DT_BF16, st));
  THIP(launch_ln_fwd(h, s->T, C, eps, s->pp(b.ln2g), s->pp(b.ln2b), a2, st2, st));
  TCHK(linear(s, R, tseg(C, tvin(a2, C)), s->at(b.w_fc1), C, s->pp(b.fc1b), nullptr, z, nullptr,
              DT_BF16, st));
  THIP(launch_gelu_fwd(z, m, s->T * R, st));
  TCHK(linear(s, C, tseg(R, tvin(m, R)), s->at(b.w_fc2), R, s->pp(b.fc2b), h, out, out2,
              DT_BF16, st));
  return PULSE_OK;
}

// Stream plumbing of the backward pass.  With the side stream, each
// parameter gradient (weight-gradient GEMM and bias sum) is handed to it as
// soon as its output gradient exists; the caller's stream goes on with the
// data gradient.  Scratch that the side stream reads is not overwritten by
// the caller's stream before the side stream's event for it has fired.
struct BwdSync {
  pulse_tstage* s;
  hipStream_t st;     // the caller's stream
  hipStream_t work;   // where parameter gradients run: side or st
  float* red;         // their reduction buffer
  bool on_side;
  hipEvent_t last = nullptr;  // the side stream's latest recorded event
};

hipEvent_t sync_event(pulse_tstage* s) {
  if (s->sev_used == s->sev.size()) {
    hipEvent_t e;
    if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return nullptr;
    s->sev.push_back(e);
  }
  return s->sev[s->sev_used++];
}

BwdSync bwd_sync(pulse_tstage* s, hipStream_t st, bool keep_events = false) {
  BwdSync y;
  y.s = s;
  y.st = st;
  y.on_side = s->side != nullptr && !s->timing;
  y.work = y.on_side ? s->side : st;
  y.red = s->fat(y.on_side ? s->s_red2 : s->s_red);
  if (!keep_events) s->sev_used = 0;
  return y;
}

// A decoder backward left running beside its stream: `st` waits for all of
// the side stream's work so far (clear: the pending state is done with).
pulse_status tsettle(const pulse_tstage* s, hipStream_t st) {
  if (!s->join_pending) return PULSE_OK;
  THIP(hipEventRecord(s->ev_settle, s->side));
  THIP(hipStreamWaitEvent(st, s->ev_settle, 0));
  return PULSE_OK;
}

pulse_status tsettle(pulse_tstage* s, hipStream_t st, bool clear) {
  TCHK(tsettle(static_cast<const pulse_tstage*>(s), st));
  if (clear) s->join_pending = false;
  return PULSE_OK;
}

// make the side stream wait for everything enqueued on the caller's stream
pulse_status fork(BwdSync& y) {
  if (!y.on_side) return PULSE_OK;
  hipEvent_t e = sync_event(y.s);
  if (!e) return tfail(PULSE_E_HIP, "hipEventCreate failed");
  THIP(hipEventRecord(e, y.st));
  THIP(hipStreamWaitEvent(y.s->side, e, 0));
  return PULSE_OK;
}

// an event after the side stream's work so far (null without a side stream)
pulse_status mark(BwdSync& y, hipEvent_t* out) {
  *out = nullptr;
  if (!y.on_side) return PULSE_OK;
  hipEvent_t e = sync_event(y.s);
  if (!e) return tfail(PULSE_E_HIP, "hipEventCreate failed");
  THIP(hipEventRecord(e, y.s->side));
  *out = y.last = e;
  return PULSE_OK;
}

pulse_status wait_for(BwdSync& y, hipEvent_t e) {
  if (e) THIP(hipStreamWaitEvent(y.st, e, 0));
  return PULSE_OK;
}

// the caller's stream waits for all side work
pulse_status join(BwdSync& y) { return wait_for(y, y.last); }

// parameter gradients of one linear layer: bias += colsum(gy), W += gy^T in;
// with `part` the column sums come from the producer of gy as partials
// [rows][2][M]
pulse_status param_grads(BwdSync& y, int M, const Seg& in, const void* gy, float* bias,
                         const float* part = nullptr, int rows = 0) {
  TCHK(fork(y));
  if (part)
    TCHK(totals(part, rows, M, bias, y.work));
  else
    TCHK(col_sum(y.s, gy, M, bias, y.red, y.work));
  TCHK(linear_wgrad(y.s, M, in, gy, y.work));
  return PULSE_OK;
}

// dx = d(block)/dx^T dy for the block input x; parameter gradients +=
pulse_status block_bwd(BwdSync& y, SideReads& rd, int par, char* row, const TBlock& b,
                       const void* x, const void* dy, void* dx, float* dx_csum = nullptr) {
  pulse_tstage* s = y.s;
  hipStream_t st = y.st;
  const int C = s->C, R = s->R;
  const long T = s->T;
  void* a = row + b.r_a;
  const float* st1 = reinterpret_cast<const float*>(row + b.r_st1);
  void* qkv = row + b.r_qkv;
  void* o = row + b.r_o;
  void* h = row + b.r_h;
  void* a2 = row + b.r_a2;
  const float* st2 = reinterpret_cast<const float*>(row + b.r_st2);
  void* z = row + b.r_z;
  void* m = row + b.r_m;
  void* dm = s->at(s->s_dm[par]);
  void* da2 = s->at(s->s_da2);
  void* dh = s->at(s->s_dh[par]);
  void* dO = s->at(s->s_do);
  void* dqkv = s->at(s->s_dqkv[par]);
  void* da = s->at(s->s_da);
  // MLP: y = h + Fc2(GELU(Fc1(LN2(h))))
  TCHK(param_grads(y, C, tseg(R, tvin(m, R), s->gp(b.fc2W)), dy, s->gp(b.fc2b)));
  TCHK(mark(y, &rd.dy));
  TCHK(wait_for(y, rd.dm));
  TCHK(linear(s, R, tseg(C, tvin(dy, C)), s->at(b.t_fc2), C, nullptr, nullptr, dm, nullptr,
              DT_BF16, st));
  THIP(launch_gelu_bwd(dm, z, dm, T * R, st));
  TCHK(param_grads(y, R, tseg(C, tvin(a2, C), s->gp(b.fc1W)), dm, s->gp(b.fc1b)));
  TCHK(mark(y, &rd.dm));
  TCHK(linear(s, C, tseg(R, tvin(dm, R)), s->at(b.t_fc1), R, nullptr, nullptr, da2, nullptr,
              DT_BF16, st));
  TCHK(wait_for(y, rd.dh));
  float* cs_h = s->fat(s->s_cs_h[par]);
  TCHK(ln_backward(s, da2, h, st2, b.ln2g, b.ln2b, dy, dh, st, cs_h));
  // attention: h = x + Proj(MHA(LN1(x)))
  TCHK(param_grads(y, C, tseg(C, tvin(o, C), s->gp(b.projW)), dh, s->gp(b.projb), cs_h,
                   ln_bwd_blocks(T)));
  TCHK(mark(y, &rd.dh));
  TCHK(linear(s, C, tseg(C, tvin(dh, C)), s->at(b.t_proj), C, nullptr, nullptr, dO, nullptr,
              DT_BF16, st));
  TCHK(wait_for(y, rd.dqkv));
  THIP(launch_attn_bwd(qkv, o, dO, reinterpret_cast<const float*>(row + b.r_lse), s->B, s->L, C,
                       s->H, dqkv, s->fat(s->s_dsum), st));
  TCHK(param_grads(y, 3 * C, tseg(C, tvin(a, C), s->gp(b.qkvW)), dqkv, s->gp(b.qkvb)));
  TCHK(mark(y, &rd.dqkv));
  TCHK(linear(s, C, tseg(3 * C, tvin(dqkv, 3 * C)), s->at(b.t_qkv), 3 * C, nullptr, nullptr, da,
              nullptr, DT_BF16, st));
  TCHK(ln_backward(s, da, x, st1, b.ln1g, b.ln1b, dh, dx, st, dx_csum));
  return PULSE_OK;
}

// ---------------------------------------------------------------------------
// bookkeeping
// ---------------------------------------------------------------------------

int find_row(const pulse_tstage* s, int mb) {
  for (size_t i = 0; i < s->rows.size(); ++i)
    if (s->rows[i].mb == mb) return (int)i;
  return -1;
}

int free_row(const pulse_tstage* s) {
  for (size_t i = 0; i < s->rows.size(); ++i)
    if (s->rows[i].mb < 0) return (int)i;
  return -1;
}

pulse_status check_ptr(const void* p, const char* what) {
  if (!p) return tfail(PULSE_E_INVALID_ARG, "%s is NULL", what);
  if (reinterpret_cast<uintptr_t>(p) % 16)
    return tfail(PULSE_E_INVALID_ARG, "%s is not 16-byte aligned", what);
  return PULSE_OK;
}

pulse_status need_ready(const pulse_tstage* s) {
  if (s->dry) return PULSE_OK;
  if (!s->bound) return tfail(PULSE_E_NOT_BOUND, "stage has no bound parameters/workspace");
  if (!s->synced) return tfail(PULSE_E_NOT_BOUND, "pulse_tstage_sync_params has not run");
  return PULSE_OK;
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================

extern "C" {

pulse_status pulse_tstage_create(const pulse_tstage_desc* desc, pulse_tstage** out) {
  if (!out) return tfail(PULSE_E_INVALID_ARG, "out is NULL");
  *out = nullptr;
  TCHK(tvalidate(desc));
  pulse_tstage* s = new (std::nothrow) pulse_tstage();
  if (!s) return tfail(PULSE_E_INVALID_ARG, "out of host memory");
  s->d = *desc;
  s->dry = (desc->flags & PULSE_FLAG_DRY_RUN) != 0;
  s->B = desc->batch;
  s->L = desc->tokens;
  s->C = desc->width;
  s->H = desc->heads;
  s->R = desc->mlp_ratio * desc->width;
  s->T = (long)s->B * s->L;
  // each image's tokens as one row of L pixels: the weight-gradient kernel
  // steps its pixel coordinates 64 at a time, one wrap per row
  s->geo = Geo{s->B, 1, s->L};
  const int ct = env_or("PULSE_TCONV_TILE", -1);
  s->conv_tile_force = (ct >= 0 && ct <= TILE2_CONV_LAST) ? ct : -1;
  s->conv_ks_cap = std::max(1, std::min(16, env_or("PULSE_TCONV_KSPLIT_MAX", 16)));
  s->wgrad_tile_force = env_or("PULSE_TWGRAD_TILE", -1);
  build_layout(s);
  s->rows.resize(desc->max_inflight);
  *out = s;
  return PULSE_OK;
}

void pulse_tstage_destroy(pulse_tstage* s) {
  if (!s) return;
  // work a decoder backward left on the side stream ends before its events go
  if (s->side) (void)hipStreamSynchronize(s->side);
  if (s->ev_settle) (void)hipEventDestroy(s->ev_settle);
  for (hipEvent_t e : s->ev_pool) (void)hipEventDestroy(e);
  for (hipEvent_t e : s->sev) (void)hipEventDestroy(e);
  if (s->side) (void)hipStreamDestroy(s->side);
  delete s;
}

pulse_status pulse_tstage_sizes(const pulse_tstage* s, int64_t* n_params, size_t* ws_bytes) {
  if (!s) return tfail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (n_params) *n_params = s->n_params;
  if (ws_bytes) *ws_bytes = s->dry ? 0 : s->ws_bytes;
  return PULSE_OK;
}

pulse_status pulse_tstage_param_layout(const pulse_tstage* s, int32_t idx, char name[64],
                                       int64_t* offset, int32_t shape[4]) {
  if (!s) return tfail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (idx == -1) {
    if (!offset) return tfail(PULSE_E_INVALID_ARG, "offset is NULL");
    *offset = (int64_t)s->params.size();
    return PULSE_OK;
  }
  if (idx < 0 || idx >= (int)s->params.size())
    return tfail(PULSE_E_INVALID_ARG, "parameter index %d out of range", idx);
  const TParam& p = s->params[idx];
  if (name) {
    std::strncpy(name, p.name.c_str(), 63);
    name[63] = 0;
  }
  if (offset) *offset = p.off;
  if (shape)
    for (int i = 0; i < 4; ++i) shape[i] = p.shape[i];
  return PULSE_OK;
}

pulse_status pulse_tstage_bind(pulse_tstage* s, const float* params, float* grads, void* ws,
                               size_t ws_bytes) {
  if (!s) return tfail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (s->dry) return tfail(PULSE_E_STATE, "a dry-run stage binds no memory");
  if (!params || !grads || !ws) return tfail(PULSE_E_INVALID_ARG, "NULL pointer in bind");
  if (reinterpret_cast<uintptr_t>(ws) % 256 || reinterpret_cast<uintptr_t>(params) % 16 ||
      reinterpret_cast<uintptr_t>(grads) % 16)
    return tfail(PULSE_E_INVALID_ARG, "workspace must be 256-byte, params/grads 16-byte aligned");
  if (ws_bytes < s->ws_bytes)
    return tfail(PULSE_E_INVALID_ARG, "workspace %zu bytes < required %zu", ws_bytes, s->ws_bytes);
  if (pulse_tstage_inflight(s) > 0)
    return tfail(PULSE_E_STATE, "cannot rebind with microbatches in flight");
  if (!s->side && env_or("PULSE_SERIAL", 0) == 0) {
    // default priority, no implicit synchronisation with the null stream
    THIP(hipStreamCreateWithFlags(&s->side, hipStreamNonBlocking));
    THIP(hipEventCreateWithFlags(&s->ev_settle, hipEventDisableTiming));
  }
  s->prm = params;
  s->grd = grads;
  s->ws = static_cast<char*>(ws);
  s->bound = true;
  s->synced = false;
  return PULSE_OK;
}

pulse_status pulse_tstage_sync_params(pulse_tstage* s, void* stream) {
  if (!s) return tfail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (s->dry) {
    s->synced = true;
    return PULSE_OK;
  }
  if (!s->bound) return tfail(PULSE_E_NOT_BOUND, "stage is not bound");
  hipStream_t st = static_cast<hipStream_t>(stream);
  TCHK(tsettle(s, st, true));
  const int C = s->C, R = s->R;
  for (auto* v : {&s->eb, &s->db})
    for (const TBlock& b : *v) {
      THIP(launch_convert_rows(s->pp(b.qkvW), 3 * C, C, s->at(b.w_qkv), C, 0, DT_BF16, st));
      THIP(launch_transpose(s->pp(b.qkvW), 3 * C, C, s->at(b.t_qkv), DT_BF16, st));
      THIP(launch_convert_rows(s->pp(b.projW), C, C, s->at(b.w_proj), C, 0, DT_BF16, st));
      THIP(launch_transpose(s->pp(b.projW), C, C, s->at(b.t_proj), DT_BF16, st));
      THIP(launch_convert_rows(s->pp(b.fc1W), R, C, s->at(b.w_fc1), C, 0, DT_BF16, st));
      THIP(launch_transpose(s->pp(b.fc1W), R, C, s->at(b.t_fc1), DT_BF16, st));
      THIP(launch_convert_rows(s->pp(b.fc2W), C, R, s->at(b.w_fc2), R, 0, DT_BF16, st));
      THIP(launch_transpose(s->pp(b.fc2W), C, R, s->at(b.t_fc2), DT_BF16, st));
      if (b.dec) {
        THIP(launch_convert_rows(s->pp(b.skW), C, 2 * C, s->at(b.w_sk), 2 * C, 0, DT_BF16, st));
        THIP(launch_transpose(s->pp(b.skW), C, 2 * C, s->at(b.t_sk), DT_BF16, st));
      }
    }
  THIP(hipMemsetAsync(s->at(s->s_zero), 0, 256, st));
  s->synced = true;
  return PULSE_OK;
}

pulse_status pulse_tstage_forward(pulse_tstage* s, pulse_half half, int32_t mb, const void* in,
                                  void* out, void* stream) {
  if (!s) return tfail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (half != PULSE_ENC && half != PULSE_DEC) return tfail(PULSE_E_INVALID_ARG, "bad half");
  if (mb < 0) return tfail(PULSE_E_INVALID_ARG, "microbatch id must be >= 0");
  TCHK(need_ready(s));
  if (!s->dry) {
    TCHK(check_ptr(in, "in"));
    TCHK(check_ptr(out, "out"));
  }
  int r = find_row(s, mb);
  if (half == PULSE_ENC) {
    if (r >= 0) return tfail(PULSE_E_STATE, "microbatch %d already ran its encoder forward", mb);
    r = free_row(s);
    if (r < 0)
      return tfail(PULSE_E_CACHE_FULL, "more than max_inflight=%d microbatches in flight",
                   s->d.max_inflight);
  } else {
    if (r < 0 || s->rows[r].state != T_ENC_FWD)
      return tfail(PULSE_E_STATE, "decoder forward of microbatch %d needs its encoder forward",
                   mb);
  }
  if (!s->dry) {
    hipStream_t st = static_cast<hipStream_t>(stream);
    TCHK(tsettle(s, st, true));
    char* row = s->row(r);
    const size_t act = (size_t)s->T * s->C * 2;
    const int ne = s->d.n_enc;
    if (half == PULSE_ENC) {
      THIP(hipMemcpyAsync(row + s->eb[0].r_x, in, act, hipMemcpyDeviceToDevice, st));
      for (int k = 0; k < ne; ++k) {
        const void* x = k == 0 ? row + s->eb[0].r_x : row + s->row_slot[k - 1];
        TCHK(block_fwd(s, row, s->eb[k], x, row + s->row_slot[k], k == ne - 1 ? out : nullptr,
                       st));
      }
    } else {
      const int C = s->C;
      THIP(hipMemcpyAsync(row + s->db[0].r_v, in, act, hipMemcpyDeviceToDevice, st));
      for (int k = 0; k < s->d.n_dec; ++k) {
        const TBlock& b = s->db[k];
        const void* skip = row + s->row_slot[ne - 1 - k];
        TCHK(linear(s, C, tseg(2 * C, tvin2(row + b.r_v, C, skip, C)), s->at(b.w_sk), 2 * C,
                    s->pp(b.skb), nullptr, row + b.r_x, nullptr, DT_BF16, st));
        void* y = k == s->d.n_dec - 1 ? out : row + s->db[k + 1].r_v;
        TCHK(block_fwd(s, row, b, row + b.r_x, y, nullptr, st));
      }
    }
  }
  s->rows[r].mb = mb;
  s->rows[r].state = half == PULSE_ENC ? T_ENC_FWD : T_DEC_FWD;
  return PULSE_OK;
}

pulse_status pulse_tstage_backward(pulse_tstage* s, pulse_half half, int32_t mb,
                                   const void* dout, void* din, void* stream) {
  if (!s) return tfail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (half != PULSE_ENC && half != PULSE_DEC) return tfail(PULSE_E_INVALID_ARG, "bad half");
  TCHK(need_ready(s));
  if (!s->dry) {
    TCHK(check_ptr(dout, "dout"));
    TCHK(check_ptr(din, "din"));
  }
  const int r = find_row(s, mb);
  const int want = half == PULSE_DEC ? T_DEC_FWD : T_DEC_BWD;
  if (r < 0 || s->rows[r].state != want)
    return tfail(PULSE_E_STATE, "%s backward of microbatch %d out of order",
                 half == PULSE_DEC ? "decoder" : "encoder", mb);
  if (!s->dry) {
    hipStream_t st = static_cast<hipStream_t>(stream);
    char* row = s->row(r);
    const int C = s->C, ne = s->d.n_enc, nd = s->d.n_dec;
    const long T = s->T;
    const bool carry = half == PULSE_ENC && s->join_pending && s->pending_mb == mb &&
                       s->pending_st == st && s->side && !s->timing;
    if (!carry) TCHK(tsettle(s, st, true));
    BwdSync y = bwd_sync(s, st, carry);
    SideReads rds[2];
    if (carry) {
      // The decoder's last parameter-gradient work may still run on the side
      // stream.  It read the dy buffers last in its final fc2 weight
      // gradient, which this stream waits for before writing them; its dm,
      // dh, dqkv and column-partial buffers are guarded per parity by the
      // carried events; its skip-linear buffers this call does not write.
      rds[0] = s->pending_rds[0];
      rds[1] = s->pending_rds[1];
      TCHK(wait_for(y, s->pending_dy));
      s->join_pending = false;
    }
    hipEvent_t dec_dy_read = nullptr;
    if (half == PULSE_DEC) {
      const void* dy = dout;
      hipEvent_t dy_read = nullptr;  // the side stream has read the previous block's dy
      for (int k = nd - 1; k >= 0; --k) {
        const TBlock& b = s->db[k];
        SideReads& rd = rds[k & 1];
        void* dsx = s->at(s->s_dsx[k & 1]);
        TCHK(wait_for(y, rd.dsx));
        float* cs_x = s->fat(s->s_cs_x[k & 1]);
        TCHK(block_bwd(y, rd, k & 1, row, b, row + b.r_x, dy, dsx, cs_x));
        // skip linear over [v || skip]
        const int slot = ne - 1 - k;
        const void* skip = row + s->row_slot[slot];
        TCHK(param_grads(y, C, tseg(2 * C, tvin2(row + b.r_v, C, skip, C), s->gp(b.skW)), dsx,
                         s->gp(b.skb), cs_x, ln_bwd_blocks(s->T)));
        TCHK(mark(y, &rd.dsx));
        void* dv = k == 0 ? din : s->at(s->s_dy[k & 1]);
        // dv's buffer held the dy of block k + 1, which the side stream reads
        TCHK(wait_for(y, dy_read));
        dy_read = rd.dy;
        const char* tsk = s->at(b.t_sk);
        TCHK(linear(s, C, tseg(C, tvin(dsx, C)), tsk, C, nullptr, nullptr, dv, nullptr, DT_BF16,
                    st));
        TCHK(linear(s, C, tseg(C, tvin(dsx, C)), tsk + (size_t)C * C * 2, C, nullptr, nullptr,
                    row + s->row_sgrad[slot], nullptr, DT_F32, st));
        dy = dv;
      }
      dec_dy_read = dy_read;
    } else {
      const void* g = dout;
      for (int k = ne - 1; k >= 0; --k) {
        const TBlock& b = s->eb[k];
        // the gradient reaching x_k: from its encoder consumer and from the
        // buffered skip gradient of its decoder consumer
        SideReads& rd = rds[k & 1];
        void* dy = s->at(s->s_dy[0]);
        // the previous block's fc2 parameter gradient read this buffer
        TCHK(wait_for(y, rds[(k + 1) & 1].dy));
        THIP(launch_add_cast(g, DT_BF16, reinterpret_cast<const float*>(row + s->row_sgrad[k]),
                             dy, DT_BF16, T * C, st));
        const void* x = k == 0 ? row + b.r_x : row + s->row_slot[k - 1];
        void* dx = k == 0 ? din : s->at(s->s_dy[1]);
        TCHK(block_bwd(y, rd, k & 1, row, b, x, dy, dx));
        g = dx;
      }
    }
    if (half == PULSE_DEC && s->overlap_bwd && y.on_side) {
      // the side stream's remaining work joins at the next call
      s->join_pending = true;
      s->pending_mb = mb;
      s->pending_st = st;
      s->pending_rds[0] = rds[0];
      s->pending_rds[1] = rds[1];
      s->pending_dy = dec_dy_read;
    } else {
      TCHK(join(y));
    }
  }
  if (half == PULSE_DEC) {
    s->rows[r].state = T_DEC_BWD;
  } else {
    s->rows[r] = TRow();
  }
  return PULSE_OK;
}

pulse_status pulse_tstage_skip_grad(const pulse_tstage* s, int32_t mb, int32_t slot, float* dst,
                                    void* stream) {
  if (!s) return tfail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (slot < 0 || slot >= s->d.n_enc) return tfail(PULSE_E_INVALID_ARG, "slot out of range");
  const int r = find_row(s, mb);
  if (r < 0 || s->rows[r].state != T_DEC_BWD)
    return tfail(PULSE_E_CACHE_MISS, "no buffered skip gradient for microbatch %d", mb);
  if (s->dry) return PULSE_OK;
  TCHK(check_ptr(dst, "dst"));
  TCHK(tsettle(s, static_cast<hipStream_t>(stream)));
  THIP(hipMemcpyAsync(dst, s->row(r) + s->row_sgrad[slot], (size_t)s->T * s->C * 4,
                      hipMemcpyDeviceToDevice, static_cast<hipStream_t>(stream)));
  return PULSE_OK;
}

pulse_status pulse_tstage_release(pulse_tstage* s, int32_t mb) {
  if (!s) return tfail(PULSE_E_INVALID_ARG, "stage is NULL");
  const int r = find_row(s, mb);
  if (r >= 0) s->rows[r] = TRow();
  return PULSE_OK;
}

pulse_status pulse_tstage_reset(pulse_tstage* s) {
  if (!s) return tfail(PULSE_E_INVALID_ARG, "stage is NULL");
  for (TRow& r : s->rows) r = TRow();
  return PULSE_OK;
}

int32_t pulse_tstage_inflight(const pulse_tstage* s) {
  if (!s) return 0;
  int n = 0;
  for (const TRow& r : s->rows) n += r.mb >= 0;
  return n;
}

pulse_status pulse_tstage_overlap_bwd(pulse_tstage* s, int32_t enable) {
  if (!s) return tfail(PULSE_E_INVALID_ARG, "stage is NULL");
  s->overlap_bwd = enable != 0;
  return PULSE_OK;
}

pulse_status pulse_tstage_flush(pulse_tstage* s, void* stream) {
  if (!s) return tfail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (s->dry) return PULSE_OK;
  return tsettle(s, static_cast<hipStream_t>(stream), true);
}

pulse_status pulse_tstage_timing(pulse_tstage* s, int32_t enable) {
  if (!s) return tfail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (s->join_pending) {  // timed calls keep everything on the caller's stream
    THIP(hipStreamSynchronize(s->side));
    s->join_pending = false;
  }
  s->timing = enable != 0;
  s->timed.clear();
  s->ev_used = 0;
  return PULSE_OK;
}

pulse_status pulse_tstage_timing_read(pulse_tstage* s, int64_t* launches, double* ms,
                                      double* flops, double* bytes) {
  if (!s) return tfail(PULSE_E_INVALID_ARG, "stage is NULL");
  double tms = 0.0, tf = 0.0, tb = 0.0;
  for (const TTimed& t : s->timed) {
    THIP(hipEventSynchronize(t.b));
    float x = 0.f;
    THIP(hipEventElapsedTime(&x, t.a, t.b));
    tms += x;
    tf += t.flops;
    tb += t.bytes;
  }
  if (launches) *launches = (int64_t)s->timed.size();
  if (ms) *ms = tms;
  if (flops) *flops = tf;
  if (bytes) *bytes = tb;
  return PULSE_OK;
}

double pulse_tstage_flops(const pulse_tstage* s) {
  if (!s) return 0.0;
  const double T = (double)s->T, C = s->C, R = s->R, L = s->L;
  // per block: forward GEMMs 2T(3C^2 + C^2 + 2RC), three times with the
  // data and weight gradients; attention 4TLC forward, 8TLC backward
  const double blk = 3.0 * 2.0 * T * (4.0 * C * C + 2.0 * R * C) + 12.0 * T * L * C;
  const double skip = 3.0 * 2.0 * T * (2.0 * C) * C;
  return (s->d.n_enc + s->d.n_dec) * blk + s->d.n_dec * skip;
}

}  // extern "C"
