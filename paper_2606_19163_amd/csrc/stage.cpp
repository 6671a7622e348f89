// Host side of the stage library: descriptor validation, parameter and
// workspace layout, the skip cache and per-microbatch bookkeeping, and the
// kernel sequence of every forward / backward half.  Implements
// include/pulse_stage.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "error.hpp"
#include "kernels.hpp"
#include "pulse_stage.h"

using namespace pulse;

namespace {

thread_local std::string g_err;

pulse_status fail(pulse_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

#define HIPCHK(expr)                                                                   \
  do {                                                                                 \
    hipError_t e_ = (expr);                                                            \
    if (e_ != hipSuccess)                                                              \
      return fail(PULSE_E_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));         \
  } while (0)

constexpr int MAX_SLOTS = 64;

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

enum RowState { R_FRESH = 1, R_ENC_FWD = 2, R_DEC_FWD = 3, R_DEC_BWD = 4 };

struct ParamInfo {
  std::string name;
  int64_t off;
  int32_t shape[4];
  int64_t numel;
};

// Offsets of one GroupNorm's saved statistics inside a row.
struct GnSave {
  size_t mean, rstd, scale, shift;
};

struct Block {
  bool dec;
  int cin, cout, c0;  // c0: channels of the first source (dec: c_up)
  int slot;           // enc: skip_slot_out, dec: skip_slot_in
  bool conv_sc;
  // parameter offsets (elements)
  int64_t W1, b1, Wl, bl, g1, be1, g2, be2, W2, b2, Ws, bs;
  // compute copies of the weights (workspace byte offsets)
  size_t wf1, wf2, wd1, wd2, wsd, bias2;
  int ldb2;
  // per-row saved tensors (byte offsets inside a row)
  size_t a1_0, a1_1, h1, a2, out_saved;
  GnSave gn1, gn2;
};

struct Row {
  int mb = -1;
  int state = 0;
  bool enc_done = false;
  uint8_t act[MAX_SLOTS] = {};
  uint8_t grad[MAX_SLOTS] = {};
};

struct TimedLaunch {
  hipEvent_t a, b;
  double flops, bytes;
};

}  // namespace

pulse_status pulse::set_last_error(pulse_status s, const char* msg) {
  g_err = msg;
  return s;
}

// Side-stream progress markers of one backward call: block k records w2
// after its conv2 / shortcut parameter work (the last read of its dout) and
// w1 after its conv1 weight gradient (the last read of its dh1); buffers
// alternate between consecutive blocks, so block k waits for the marker of
// the block that used the same buffer before it.
struct BwdSync {
  bool w2[2] = {false, false}, w1[2] = {false, false};
};

struct pulse_stage {
  // descriptor
  pulse_stage_desc d{};
  std::vector<pulse_enc_block> enc;
  std::vector<pulse_dec_block> dec;
  bool dry = false;
  int dtype = DT_F32;
  size_t esz = 4;
  bool k64 = false;     // every channel count is a multiple of 64
  int conv_tile_force = -1, wgrad_tile_force = -1;  // tuning overrides (env)
  bool no_gnb = false;  // PULSE_NO_GNB: GroupNorm-backward sums by their own pass
  int conv_ksplit_cap = 16;  // largest conv K split (env PULSE_CONV_KSPLIT_MAX)
  Geo geo{};
  long P = 0;
  int G = 1;
  float eps = 1e-5f;
  int D = 0;
  // parameters
  std::vector<ParamInfo> params;
  int64_t n_params = 0;
  std::vector<Block> eb, db;
  // slots
  int n_slots = 0;
  int slot_ch[MAX_SLOTS];
  int slot_reader[MAX_SLOTS];   // decoder block index or -1
  int slot_producer[MAX_SLOTS]; // encoder block index, -2 = stage input, -1 = none
  // workspace layout
  size_t ws_bytes = 0, off_rows = 0, row_size = 0, off_scratch = 0;
  size_t row_act[MAX_SLOTS], row_grad[MAX_SLOTS];
  size_t row_temb[2] = {0, 0}, row_xin = 0, row_u = 0;
  size_t s_da = 0, s_dxs = 0, s_dh1[2] = {0, 0}, s_g[2] = {0, 0}, s_part = 0, s_red = 0, s_coef = 0,
         s_pi = 0, s_e = 0, s_zero = 0;
  size_t part_cap = 0;   // weight-gradient split partials (elements)
  size_t kpart_cap = 0;  // conv K-split partials (elements)
  size_t s_kpart = 0, s_red2 = 0;
  size_t s_chp[2] = {0, 0};  // per-chunk channel sums of dh1 (GN2 backward), by block parity
  int cmax = 0;              // widest channel count of any block
  size_t red_cap = 0;        // floats in each reduction buffer
  // side stream: the weight-gradient GEMMs of the backward pass run on it,
  // concurrently with the data-gradient chain on the caller's stream
  hipStream_t side = nullptr;
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  // ev_fork was recorded by the completion of the last kernel enqueued on
  // the caller's stream (the next fork needs no marker of its own)
  bool fork_attached = false;
  // overlapped decoder backward (pulse_stage_overlap_bwd): a decoder
  // backward may return with its last parameter-gradient work still on the
  // side stream; the next call joins it, except an encoder backward of the
  // same microbatch on the same stream, which continues beside it
  bool overlap_bwd = false;
  bool join_pending = false;
  int32_t pending_mb = -1;
  hipStream_t pending_st = nullptr;
  BwdSync sy_pending;  // the decoder call's markers, carried into the encoder call
  int par_pending = 0;  // parity of the decoder call's last block
  hipEvent_t ev_w2[2] = {nullptr, nullptr}, ev_w1[2] = {nullptr, nullptr};
  // Every call shares the scratch buffers.  The stream of the last call that
  // enqueued work and an event recorded at its end let a call on another
  // stream wait for it first.
  hipStream_t last_st = nullptr;
  hipEvent_t ev_last = nullptr;
  bool have_last = false;
  // binding
  const float* prm = nullptr;
  float* grd = nullptr;
  char* ws = nullptr;
  bool bound = false;
  bool synced = false;
  std::vector<Row> rows;
  // timing of the implicit-GEMM conv launches
  bool timing = false;
  std::vector<TimedLaunch> timed;
  std::vector<hipEvent_t> ev_pool;
  size_t ev_used = 0;

  char* row_base(int r) const { return ws + off_rows + (size_t)r * row_size; }
  void* scratch(size_t off) const { return ws + off_scratch + off; }
  float* sf(size_t off) const { return reinterpret_cast<float*>(scratch(off)); }
  // Scratch of the forward pass (GroupNorm partial sums, timestep
  // projections, conv K-split partials): the bound workspace's regions for
  // every call but pulse_stage_forward_static, which points fwd_base at the
  // library's static device array and the offsets at a compact layout.
  char* fwd_base = nullptr;
  size_t f_red = 0, f_e = 0, f_kpart = 0, f_kcap = 0;
  size_t fs_red = 0, fs_e = 0, fs_kpart = 0, fs_kcap = 0, fs_bytes = 0;  // compact layout
  float* fwd(size_t off) const { return reinterpret_cast<float*>(fwd_base + off); }
  void use_workspace_scratch() {
    fwd_base = ws + off_scratch;
    f_red = s_red;
    f_e = s_e;
    f_kpart = s_kpart;
    f_kcap = kpart_cap;
  }
  const float* pp(int64_t off) const { return prm + off; }
  float* gp(int64_t off) const { return off < 0 ? nullptr : grd + off; }
};

namespace {

// ---------------------------------------------------------------------------
// layout
// ---------------------------------------------------------------------------

int64_t add_param(pulse_stage* s, const std::string& name, std::initializer_list<int> shape) {
  ParamInfo p;
  p.name = name;
  p.off = s->n_params;
  int i = 0;
  p.numel = 1;
  for (int x : shape) {
    p.shape[i++] = x;
    p.numel *= x;
  }
  for (; i < 4; ++i) p.shape[i] = 0;
  s->params.push_back(p);
  s->n_params += (p.numel + 63) / 64 * 64;
  return p.off;
}

void layout_params(pulse_stage* s, Block& b, const std::string& pre) {
  b.W1 = add_param(s, pre + "W1", {b.cout, 3, 3, b.cin});
  b.b1 = add_param(s, pre + "b1", {b.cout});
  b.Wl = add_param(s, pre + "Wl", {b.cout, s->D});
  b.bl = add_param(s, pre + "bl", {b.cout});
  b.g1 = add_param(s, pre + "g1", {b.cin});
  b.be1 = add_param(s, pre + "be1", {b.cin});
  b.g2 = add_param(s, pre + "g2", {b.cout});
  b.be2 = add_param(s, pre + "be2", {b.cout});
  b.W2 = add_param(s, pre + "W2", {b.cout, 3, 3, b.cout});
  b.b2 = add_param(s, pre + "b2", {b.cout});
  if (b.conv_sc) {
    b.Ws = add_param(s, pre + "Ws", {b.cout, b.cin});
    b.bs = add_param(s, pre + "bs", {b.cout});
  } else {
    b.Ws = b.bs = -1;
  }
}

size_t act_bytes(const pulse_stage* s, int C) { return (size_t)s->P * C * s->esz; }

void layout_gn(const pulse_stage* s, GnSave& g, size_t& off, int C) {
  g.mean = off;
  off += align256((size_t)s->geo.B * s->G * 4);
  g.rstd = off;
  off += align256((size_t)s->geo.B * s->G * 4);
  g.scale = off;
  off += align256((size_t)s->geo.B * C * 4);
  g.shift = off;
  off += align256((size_t)s->geo.B * C * 4);
}

// Tile shape of a conv-mode GEMM with N output columns (a Tile2 value on
// the LDS-DMA path, a Tile value otherwise).
int conv_tile(const pulse_stage* s, int N) {
  if (s->dtype == DT_F32) return TILE_64x64_F32;
  if (!s->k64) return TILE_128x128_K32;
  if (s->conv_tile_force >= 0) return s->conv_tile_force;
  return N % 160 == 0 ? TILE2_C128x160 : TILE2_C128x128;
}

// Tile shape of a weight-gradient GEMM (M output channels, N columns).
int wgrad_tile(const pulse_stage* s, int M, int N) {
  if (s->dtype == DT_F32) return TILE_64x64_F32;
  if (!s->k64) return TILE_128x128_K32;
  if (s->wgrad_tile_force >= 0) return s->wgrad_tile_force;
  (void)N;
  return M % 320 == 0 ? TILE2_W320x128 : TILE2_W128x128;
}

// bf16 with every channel count a multiple of 64: the LDS-DMA kernels
bool uses_v2(const pulse_stage* s) { return s->dtype == DT_BF16 && s->k64; }

TileInfo info_of(const pulse_stage* s, int tile) {
  return uses_v2(s) ? tile2_info(tile) : tile_info(tile);
}

// K splits of a conv-mode GEMM on the LDS-DMA path: enough blocks for two
// per CU (the tile's occupancy), each split keeping at least 4 K-steps.
int conv_ksplit(const pulse_stage* s, int tile, int N, int K) {
  if (!uses_v2(s)) return 1;
  const TileInfo ti = info_of(s, tile);
  const long tiles = ((s->P + ti.bm - 1) / ti.bm) * ((N + ti.bn - 1) / ti.bn);
  const long want = 512;
  if (tiles >= want) return 1;
  long ks = (want + tiles - 1) / tiles;
  ks = std::min(ks, std::max(1L, (long)(K / ti.bk) / 4));
  return (int)std::min(ks, (long)s->conv_ksplit_cap);
}

// Pixel split of a weight-gradient GEMM.  With s splits the grid holds
// tiles * s blocks of K / s pixels each; blocks run in ceil(tiles * s /
// slots) rounds, and every split adds an fp32 partial of M x N that is
// written once and read once by the finalize, which then reads and writes
// the fp32 gradient.  The split count minimises
//   rounds(s) * T_tile / s + bytes(s) * M * N / HBM
// where T_tile is one tile's whole-K time at a nominal per-CU rate and
// bytes(s) = 8 s + 8; on the LDS-DMA path one split adds its tile into the
// gradient in the GEMM epilogue (no partial, no finalize): bytes(1) = 8.
int pick_splits(const pulse_stage* s, int tile, int M, int N, int& kchunk) {
  const TileInfo ti = info_of(s, tile);
  const long tiles = (long)((M + ti.bm - 1) / ti.bm) * ((N + ti.bn - 1) / ti.bn);
  const long per_cu = ti.per_cu > 0 ? std::min(ti.per_cu, 2) : (ti.bm * ti.bn <= 128 * 128 ? 2 : 1);
  const long slots = 256L * per_cu;  // resident blocks
  const double t_tile = 2.0 * ti.bm * ti.bn * (double)s->P / 3.0e12;  // s, per CU
  const double t_elem = (double)M * N / 4.0e12;                       // s per byte per element
  const long maxs = std::max(1L, (long)(s->P / (4 * ti.bk)));          // >= 4 K-steps each
  long best = 1;
  double best_t = 1e30;
  for (long sp = 1; sp <= std::min(maxs, 256L); ++sp) {
    const long rounds = (tiles * sp + slots - 1) / slots;
    const double bytes = sp == 1 && uses_v2(s) ? 8.0 : 8.0 * sp + 8.0;
    const double t = rounds * t_tile / sp + bytes * t_elem;
    if (t < best_t * 0.999) {
      best_t = t;
      best = sp;
    }
  }
  long kc = (s->P + best - 1) / best;
  kc = (kc + ti.bk - 1) / ti.bk * ti.bk;
  kchunk = (int)kc;
  // the kernel derives the split count from the grid: keep it exact
  return (int)((s->P + kc - 1) / kc);
}

// Weight-gradient work split: uniform pixel splits of kchunk pixels
// (pick_splits); every split writes one fp32 partial of M x N.
struct WgradPlan {
  int splits = 1, kchunk = 0, slots = 1;
};

WgradPlan wgrad_plan(const pulse_stage* s, int tile, int M, int N) {
  WgradPlan w;
  w.splits = pick_splits(s, tile, M, N, w.kchunk);
  w.slots = w.splits;
  return w;
}

int env_int(const char* name, int dflt) {
  const char* v = getenv(name);
  if (!v || !*v) return dflt;
  return atoi(v);
}

pulse_status build_layout(pulse_stage* s) {
  const pulse_stage_desc& d = s->d;
  s->dtype = d.dtype == PULSE_BF16 ? DT_BF16 : DT_F32;
  s->esz = d.dtype == PULSE_BF16 ? 2 : 4;
  s->geo = Geo{d.batch, d.height, d.width};
  s->P = s->geo.pixels();
  s->G = d.groups;
  s->eps = d.eps;
  s->D = d.temb_dim;

  // blocks and parameters
  int cmax = 0;
  for (int k = 0; k < d.n_enc; ++k) {
    Block b{};
    b.dec = false;
    b.cin = s->enc[k].c_in;
    b.cout = s->enc[k].c_out;
    b.c0 = b.cin;
    b.slot = s->enc[k].skip_slot_out;
    b.conv_sc = b.cin != b.cout;
    layout_params(s, b, "enc" + std::to_string(k) + ".");
    s->eb.push_back(b);
    cmax = std::max(cmax, std::max(b.cin, b.cout));
  }
  for (int k = 0; k < d.n_dec; ++k) {
    Block b{};
    b.dec = true;
    b.cin = s->dec[k].c_up + s->dec[k].c_skip;
    b.cout = s->dec[k].c_out;
    b.c0 = s->dec[k].c_up;
    b.slot = s->dec[k].skip_slot_in;
    b.conv_sc = b.cin != b.cout;
    layout_params(s, b, "dec" + std::to_string(k) + ".");
    s->db.push_back(b);
    cmax = std::max(cmax, std::max(b.cin, b.cout));
  }

  // bf16 tiles take 64 channels per K-step when every channel count allows
  {
    bool k64 = true;
    auto chk = [&](int c) { if (c % 64) k64 = false; };
    for (auto& b : s->eb) { chk(b.cin); chk(b.cout); chk(b.c0); }
    for (auto& b : s->db) { chk(b.cin); chk(b.cout); chk(b.c0); }
    s->k64 = k64;
    // tile overrides (tuning) index Tile2; they apply on the LDS-DMA path
    const int ct = env_int("PULSE_CONV_TILE", -1), wt = env_int("PULSE_WGRAD_TILE", -1);
    s->conv_ksplit_cap = std::max(1, std::min(16, env_int("PULSE_CONV_KSPLIT_MAX", 16)));
    s->no_gnb = env_int("PULSE_NO_GNB", 0) != 0;
    const bool v2 = s->dtype == DT_BF16 && k64;
    s->conv_tile_force = (v2 && ct >= 0 && ct <= TILE2_CONV_LAST) ? ct : -1;
    s->wgrad_tile_force = (v2 && wt >= TILE2_WGRAD_FIRST && wt <= TILE2_WGRAD_LAST) ? wt : -1;
  }

  // workspace: weight copies | rows | scratch
  size_t off = 0;
  for (auto* v : {&s->eb, &s->db})
    for (auto& b : *v) {
      b.wf1 = off; off += align256((size_t)b.cout * 9 * b.cin * s->esz);
      b.ldb2 = 9 * b.cout + (b.conv_sc ? b.cin : 0);
      b.wf2 = off; off += align256((size_t)b.cout * b.ldb2 * s->esz);
      b.wd1 = off; off += align256((size_t)b.cin * 9 * b.cout * s->esz);
      b.wd2 = off; off += align256((size_t)b.cout * 9 * b.cout * s->esz);
      b.wsd = off; off += b.conv_sc ? align256((size_t)b.cin * b.cout * s->esz) : 0;
      b.bias2 = off; off += align256((size_t)b.cout * 4);
    }
  s->off_rows = off;

  // one row per in-flight microbatch
  size_t r = 0;
  for (int sl = 0; sl < s->n_slots; ++sl) {
    s->row_act[sl] = r;
    r += s->slot_ch[sl] ? align256(act_bytes(s, s->slot_ch[sl])) : 0;
    s->row_grad[sl] = r;
    r += s->slot_ch[sl] ? align256((size_t)s->P * s->slot_ch[sl] * 4) : 0;
  }
  for (int h = 0; h < 2; ++h) {
    s->row_temb[h] = r;
    r += align256((size_t)s->geo.B * s->D * s->esz);
  }
  s->row_xin = r; r += d.input_skip_slot >= 0 ? 0 : align256(act_bytes(s, s->eb[0].cin));
  s->row_u = r; r += align256(act_bytes(s, s->db[0].c0));
  for (auto* v : {&s->eb, &s->db})
    for (auto& b : *v) {
      b.a1_0 = r; r += align256(act_bytes(s, b.c0));
      b.a1_1 = r; r += b.cin > b.c0 ? align256(act_bytes(s, b.cin - b.c0)) : 0;
      b.h1 = r; r += align256(act_bytes(s, b.cout));
      b.a2 = r; r += align256(act_bytes(s, b.cout));
      b.out_saved = r; r += align256(act_bytes(s, b.cout));
      layout_gn(s, b.gn1, r, b.cin);
      layout_gn(s, b.gn2, r, b.cout);
    }
  s->row_size = align256(r);
  off += s->row_size * d.max_inflight;
  s->off_scratch = off;

  // scratch shared by all calls
  size_t sc = 0;
  const size_t fbig = align256((size_t)s->P * cmax * 4);
  s->s_da = sc; sc += fbig;
  s->s_dxs = sc; sc += fbig;
  s->s_dh1[0] = sc; sc += fbig;
  s->s_dh1[1] = sc; sc += fbig;
  s->s_g[0] = sc; sc += fbig;
  s->s_g[1] = sc; sc += fbig;
  size_t part = 0, kpart = 0, red = 0;
  for (auto* v : {&s->eb, &s->db})
    for (auto& b : *v) {
      int sp = wgrad_plan(s, wgrad_tile(s, b.cout, b.ldb2), b.cout, b.ldb2).slots;
      part = std::max(part, (size_t)sp * b.cout * b.ldb2);
      sp = wgrad_plan(s, wgrad_tile(s, b.cout, 9 * b.cin), b.cout, 9 * b.cin).slots;
      part = std::max(part, (size_t)sp * b.cout * 9 * b.cin);
      for (int c : {b.cin, b.cout}) {
        RedGrid rg = red_grid(s->geo, c);
        red = std::max(red, (size_t)s->geo.B * rg.chunks * 2 * c);
        // conv-mode K-split partials (an upper bound over the K of each launch)
        const int ks = conv_ksplit(s, conv_tile(s, c), c, 1 << 30);
        if (ks > 1) kpart = std::max(kpart, (size_t)ks * s->P * c);
      }
    }
  s->part_cap = part;
  s->s_part = sc; sc += align256(part * 4);
  s->kpart_cap = kpart;
  s->s_kpart = sc; sc += align256(kpart * 4);
  s->red_cap = red;
  s->s_red = sc; sc += align256(red * 4);
  s->s_red2 = sc; sc += align256(red * 4);  // reductions on the side stream
  for (int i = 0; i < 2; ++i) {
    s->s_chp[i] = sc;
    sc += align256(red * 4);
  }
  s->s_coef = sc; sc += align256((size_t)s->geo.B * s->G * 2 * 4);
  s->s_pi = sc; sc += align256((size_t)2 * s->geo.B * cmax * 4);
  s->cmax = cmax;
  // one timestep projection per block of the larger half
  const size_t nblk = std::max(s->eb.size(), s->db.size());
  s->s_e = sc; sc += align256(nblk * s->geo.B * cmax * 4);
  s->s_zero = sc; sc += 256;  // zero bytes read in place of out-of-image taps
  s->ws_bytes = s->off_scratch + sc;
  // the forward's scratch alone, packed (pulse_stage_forward_static), with
  // the K-split partials of the forward convs only, at their own K
  size_t fkpart = 0;
  for (auto* v : {&s->eb, &s->db})
    for (auto& b : *v) {
      const int k2 = 9 * b.cout + (b.conv_sc ? b.cin : 0);
      for (int K : {9 * b.cin, k2}) {
        const int ks = conv_ksplit(s, conv_tile(s, b.cout), b.cout, K);
        if (ks > 1) fkpart = std::max(fkpart, (size_t)ks * s->P * b.cout);
      }
    }
  size_t fs = 0;
  s->fs_red = fs; fs += align256(red * 4);
  s->fs_e = fs; fs += align256(nblk * s->geo.B * cmax * 4);
  s->fs_kpart = fs; fs += align256(fkpart * 4);
  s->fs_kcap = fkpart;
  s->fs_bytes = fs;
  return PULSE_OK;
}

pulse_status validate_desc(const pulse_stage_desc* d) {
  if (!d) return fail(PULSE_E_INVALID_ARG, "desc is NULL");
  if (d->dtype != PULSE_F32 && d->dtype != PULSE_BF16)
    return fail(PULSE_E_INVALID_ARG, "dtype %d unknown", (int)d->dtype);
  if (d->batch < 1 || d->height < 1 || d->width < 1)
    return fail(PULSE_E_SHAPE, "batch/height/width must be >= 1");
  // The conv kernels address pixels with 24-bit products and every operand
  // through a buffer range of at most 2^31 - 1 bytes.
  const long P = (long)d->batch * d->height * d->width;
  if (P >= (1L << 24)) return fail(PULSE_E_SHAPE, "batch*height*width must stay below 2^24 pixels");
  if (d->groups < 1 || d->groups > 256) return fail(PULSE_E_SHAPE, "groups must be in [1, 256]");
  if (!(d->eps >= 0.0f)) return fail(PULSE_E_SHAPE, "eps must be >= 0");
  if (d->temb_dim < 1) return fail(PULSE_E_SHAPE, "temb_dim must be >= 1");
  if (d->n_enc < 1 || d->n_dec < 1 || !d->enc || !d->dec)
    return fail(PULSE_E_SHAPE, "need at least one encoder and one decoder block");
  if (d->max_inflight < 1 || d->max_inflight > 64)
    return fail(PULSE_E_SHAPE, "max_inflight must be in [1, 64]");
  auto okc = [&](int c) { return c >= 32 && c % 32 == 0 && c % d->groups == 0 && c <= 8192; };
  for (int k = 0; k < d->n_enc; ++k) {
    const auto& b = d->enc[k];
    if (!okc(b.c_in) || !okc(b.c_out))
      return fail(PULSE_E_SHAPE, "enc[%d]: channels must be multiples of 32 and of groups", k);
    if (k > 0 && b.c_in != d->enc[k - 1].c_out)
      return fail(PULSE_E_SHAPE, "enc[%d].c_in != enc[%d].c_out", k, k - 1);
    if (b.skip_slot_out < -1 || b.skip_slot_out >= MAX_SLOTS)
      return fail(PULSE_E_SHAPE, "enc[%d].skip_slot_out out of range", k);
  }
  for (int k = 0; k < d->n_dec; ++k) {
    const auto& b = d->dec[k];
    if (!okc(b.c_up) || !okc(b.c_skip) || !okc(b.c_out) || !okc(b.c_up + b.c_skip))
      return fail(PULSE_E_SHAPE, "dec[%d]: channels must be multiples of 32 and of groups", k);
    if (b.c_up + b.c_skip == b.c_out)
      return fail(PULSE_E_SHAPE, "dec[%d]: c_up + c_skip must differ from c_out", k);
    if (k > 0 && b.c_up != d->dec[k - 1].c_out)
      return fail(PULSE_E_SHAPE, "dec[%d].c_up != dec[%d].c_out", k, k - 1);
    if (b.skip_slot_in < 0 || b.skip_slot_in >= MAX_SLOTS)
      return fail(PULSE_E_SHAPE, "dec[%d].skip_slot_in out of range", k);
  }
  if (d->input_skip_slot < -1 || d->input_skip_slot >= MAX_SLOTS)
    return fail(PULSE_E_SHAPE, "input_skip_slot out of range");
  // Every [pixels][C] tensor (activations in the stage dtype, fp32 skip
  // gradients and partial sums, counted at 4 bytes per value) and every
  // weight copy ([C_out][9 C_in (+ C_in)] in the stage dtype) must stay
  // below 2 GiB.
  const long esz = d->dtype == PULSE_F32 ? 4 : 2;
  long widest = 0, wbytes = 0;
  for (int k = 0; k < d->n_enc; ++k) {
    const auto& b = d->enc[k];
    widest = std::max(widest, (long)std::max(b.c_in, b.c_out));
    wbytes = std::max(wbytes, (long)b.c_out * (9L * b.c_out + b.c_in) * esz);
    wbytes = std::max(wbytes, (long)b.c_in * 9L * b.c_out * esz);
  }
  for (int k = 0; k < d->n_dec; ++k) {
    const auto& b = d->dec[k];
    const long cin = (long)b.c_up + b.c_skip;
    widest = std::max(widest, std::max(cin, (long)b.c_out));
    wbytes = std::max(wbytes, (long)b.c_out * 9L * cin * esz);
    wbytes = std::max(wbytes, (long)b.c_out * (9L * b.c_out + cin) * esz);
    wbytes = std::max(wbytes, cin * 9L * b.c_out * esz);
  }
  if (P * widest * 4 >= (1L << 31))
    return fail(PULSE_E_SHAPE, "a [pixels][%ld] tensor of 4-byte values reaches 2 GiB", widest);
  if (wbytes >= (1L << 31)) return fail(PULSE_E_SHAPE, "a conv weight copy reaches 2 GiB");
  return PULSE_OK;
}

pulse_status build_slots(pulse_stage* s) {
  const pulse_stage_desc& d = s->d;
  for (int i = 0; i < MAX_SLOTS; ++i) {
    s->slot_ch[i] = 0;
    s->slot_reader[i] = -1;
    s->slot_producer[i] = -1;
  }
  int n = 0;
  auto produce = [&](int slot, int ch, int who) -> pulse_status {
    if (slot < 0) return PULSE_OK;
    if (s->slot_producer[slot] != -1)
      return fail(PULSE_E_SHAPE, "skip slot %d has two producers", slot);
    s->slot_producer[slot] = who;
    s->slot_ch[slot] = ch;
    n = std::max(n, slot + 1);
    return PULSE_OK;
  };
  pulse_status st;
  if ((st = produce(d.input_skip_slot, d.enc[0].c_in, -2)) != PULSE_OK) return st;
  for (int k = 0; k < d.n_enc; ++k)
    if ((st = produce(d.enc[k].skip_slot_out, d.enc[k].c_out, k)) != PULSE_OK) return st;
  for (int k = 0; k < d.n_dec; ++k) {
    const int sl = d.dec[k].skip_slot_in;
    if (s->slot_producer[sl] == -1)
      return fail(PULSE_E_SHAPE, "dec[%d] reads skip slot %d that nothing fills", k, sl);
    if (s->slot_reader[sl] != -1)
      return fail(PULSE_E_SHAPE, "skip slot %d is read by two decoder blocks", sl);
    if (s->slot_ch[sl] != d.dec[k].c_skip)
      return fail(PULSE_E_SHAPE, "dec[%d].c_skip %d != slot %d channels %d", k,
                  d.dec[k].c_skip, sl, s->slot_ch[sl]);
    s->slot_reader[sl] = k;
  }
  s->n_slots = n;
  return PULSE_OK;
}

// ---------------------------------------------------------------------------
// rows (skip cache + per-microbatch state)
// ---------------------------------------------------------------------------

int find_row(const pulse_stage* s, int mb) {
  for (size_t i = 0; i < s->rows.size(); ++i)
    if (s->rows[i].mb == mb) return (int)i;
  return -1;
}

int free_row(const pulse_stage* s) {
  for (size_t i = 0; i < s->rows.size(); ++i)
    if (s->rows[i].mb < 0) return (int)i;
  return -1;
}

void release_row(Row& r) { r = Row(); }

bool row_empty(const pulse_stage* s, const Row& r) {
  for (int i = 0; i < s->n_slots; ++i)
    if (r.act[i] || r.grad[i]) return false;
  return true;
}

// ---------------------------------------------------------------------------
// kernel sequencing helpers
// ---------------------------------------------------------------------------

Src src_of(const void* p, int dtype, int C) { return Src{p, dtype, C}; }

VIn vin1(const void* p, int dtype, int C, const float* add = nullptr) {
  VIn v;
  v.s0 = src_of(p, dtype, C);
  v.s1 = src_of(nullptr, dtype, 0);
  v.c0 = C;
  v.C = C;
  v.add = add;
  return v;
}

VIn vin2(const void* p0, int dt0, int c0, const void* p1, int dt1, int c1) {
  VIn v;
  v.s0 = src_of(p0, dt0, c0);
  v.s1 = src_of(p1, dt1, c1);
  v.c0 = c0;
  v.C = c0 + c1;
  v.add = nullptr;
  return v;
}

VIn vnone() {
  VIn v{};
  v.s0.ptr = nullptr;
  return v;
}

hipEvent_t next_event(pulse_stage* s) {
  if (s->ev_used == s->ev_pool.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    s->ev_pool.push_back(e);
  }
  return s->ev_pool[s->ev_used++];
}

double elt_bytes(int dtype) { return dtype == DT_BF16 ? 2.0 : 4.0; }

double vin_bytes(const VIn& v, double pixels) {
  if (!v.s0.ptr) return 0.0;
  const double c0 = v.s1.ptr ? v.c0 : v.C;
  double b = pixels * c0 * elt_bytes(v.s0.dtype);
  if (v.s1.ptr) b += pixels * (v.C - v.c0) * elt_bytes(v.s1.dtype);
  if (v.add) b += pixels * v.C * 4.0;
  return b;
}

// Compulsory HBM bytes of one conv-mode launch: every input element once
// (the 3x3 taps re-read the same pixels), the weights once, the residual,
// the norm input that a launch reducing GroupNorm-backward sums reads, and
// every output written.
double conv_bytes(const pulse_stage* s, const GemmArgs& a) {
  const double P = (double)a.M;
  double b = 0.0;
  for (int i = 0; i < a.nseg; ++i) b += vin_bytes(a.seg[i].in, P);
  b += (double)a.N * a.K * elt_bytes(s->dtype);
  b += vin_bytes(a.resid, P);
  if (a.gnb) b += vin_bytes(a.gnb_x, P);
  b += P * a.N * elt_bytes(a.out_dtype) * (a.out2 ? 2.0 : 1.0);
  return b;
}

pulse_status run_conv(pulse_stage* s, GemmArgs& a, hipStream_t st, int* stats_chunks = nullptr) {
  if (stats_chunks) *stats_chunks = 0;
  const int tile = conv_tile(s, a.N);
  const int ks = conv_ksplit(s, tile, a.N, a.K);
  const int kt = a.K / info_of(s, tile).bk;
  a.ksplit = ks;
  a.ksteps = (kt + ks - 1) / ks;
  if (ks > 1) {
    a.ksplit = (kt + a.ksteps - 1) / a.ksteps;  // no empty split
    if ((size_t)a.ksplit * a.M * a.N > s->f_kcap)
      return fail(PULSE_E_SHAPE, "internal: conv partial buffer too small");
    a.part = s->fwd(s->f_kpart);
  }
  // timed launches: the implicit-GEMM kernels record the events themselves
  // at their start and completion; the register-staged path between markers
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (s->timing) {
    e0 = next_event(s);
    e1 = next_event(s);
  }
  const bool timed = e0 && e1;
  const bool on_kernel = timed && uses_v2(s);
  if (timed && !on_kernel) HIPCHK(hipEventRecord(e0, st));
  // Output statistics, or the GroupNorm-backward sums, from the conv: its
  // epilogue without a K split (whole tiles per image); with a K split the
  // statistics (not the backward sums, which measured slower there) from
  // the finalize on the reduction grid; with room in the reduction buffer.
  // Otherwise the caller's GroupNorm computes them itself (stats_chunks
  // stays 0).
  const bool want = (a.stats || a.gnb) && stats_chunks && uses_v2(s) &&
                    !(a.gnb && s->no_gnb);
  bool red_fin = false;
  if (want && a.ksplit == 1) {
    const int bm = info_of(s, tile).bm;
    const long rows = s->geo.hw() % bm == 0 ? (long)s->geo.B * (s->geo.hw() / bm) : 0;
    if (rows > 0 && (size_t)rows * 2 * a.N <= s->red_cap)
      *stats_chunks = s->geo.hw() / bm;
  } else if (want && a.stats && a.N % 8 == 0 && a.ldo == a.N && a.out_dtype == DT_BF16) {
    const RedGrid rg = red_grid(s->geo, a.N);
    if ((size_t)s->geo.B * rg.chunks * 2 * a.N <= s->red_cap) {
      *stats_chunks = rg.chunks;
      red_fin = true;
    }
  }
  if (!stats_chunks || *stats_chunks == 0) {
    a.stats = nullptr;
    a.gnb = nullptr;
  }
  if (red_fin) {
    GemmArgs k = a;  // the GEMM alone; the finalize below reduces
    k.stats = nullptr;
    k.gnb = nullptr;
    k.skip_finalize = 1;
    HIPCHK(launch_conv2(k, tile, st, on_kernel ? e0 : nullptr, nullptr));
    HIPCHK(launch_splitk_finalize_stats(a, red_grid(s->geo, a.N), st,
                                        on_kernel ? e1 : nullptr));
  } else if (uses_v2(s)) {
    HIPCHK(launch_conv2(a, tile, st, on_kernel ? e0 : nullptr, on_kernel ? e1 : nullptr));
  } else {
    HIPCHK(launch_conv(a, tile, st));
  }
  if (timed) {
    if (!on_kernel) HIPCHK(hipEventRecord(e1, st));
    s->timed.push_back(TimedLaunch{e0, e1, 2.0 * (double)a.M * a.N * a.K, conv_bytes(s, a)});
  }
  return PULSE_OK;
}

GemmArgs gemm_base(const pulse_stage* s) {
  GemmArgs a;
  std::memset(&a, 0, sizeof a);
  a.g = s->geo;
  a.resid = vnone();
  a.gy = vnone();
  return a;
}

Seg seg3(int begin, int C, const VIn& in, float* grad = nullptr) {
  Seg g;
  g.begin = begin;
  g.end = begin + 9 * C;
  g.taps = 9;
  g.C = C;
  g.in = in;
  g.grad = grad;
  return g;
}

Seg seg1(int begin, int C, const VIn& in, float* grad = nullptr) {
  Seg g;
  g.begin = begin;
  g.end = begin + C;
  g.taps = 1;
  g.C = C;
  g.in = in;
  g.grad = grad;
  return g;
}

// forward conv: out[P][N] = sum_seg conv(seg) (+bias, +rowvec, +resid)
// With `stats`, the output's GroupNorm partial sums come from the conv's
// epilogue when the kernel can produce them: *stats_chunks receives their
// chunks per image, or 0 when they were not computed.
// The GroupNorm+SiLU backward sums a data-gradient conv can produce for the
// GroupNorm whose output gradient it computes (see GemmArgs::gnb).
struct GnbReq {
  float* partial;
  VIn x;
  const float *scale, *shift, *mean, *rstd;
};

pulse_status conv_fwd(pulse_stage* s, int N, std::initializer_list<Seg> segs, const void* W,
                      int ldb, const float* bias, const float* rowvec, const VIn& resid,
                      void* out, void* out2, int out_dtype, hipStream_t st,
                      float* stats = nullptr, int* stats_chunks = nullptr,
                      const GnbReq* gnb = nullptr) {
  GemmArgs a = gemm_base(s);
  a.M = (int)s->P;
  a.N = N;
  int k = 0;
  for (const Seg& g : segs) {
    a.seg[a.nseg++] = g;
    k = g.end;
  }
  a.K = k;
  a.Bw = W;
  a.ldb = ldb;
  a.bias = bias;
  a.rowvec = rowvec;
  a.resid = resid;
  a.out = out;
  a.out2 = out2;
  a.out_dtype = out_dtype;
  a.ldo = N;
  a.stats = stats;
  if (gnb) {
    a.gnb = gnb->partial;
    a.gnb_x = gnb->x;
    a.gnb_scale = gnb->scale;
    a.gnb_shift = gnb->shift;
    a.gnb_mean = gnb->mean;
    a.gnb_rstd = gnb->rstd;
    a.gnb_G = s->G;
  }
  return run_conv(s, a, st, stats_chunks);
}

pulse_status wgrad(pulse_stage* s, int M, std::initializer_list<Seg> segs, const VIn& gy,
                   hipStream_t st) {
  GemmArgs a = gemm_base(s);
  a.M = M;
  int n = 0;
  for (const Seg& g : segs) {
    a.seg[a.nseg++] = g;
    n = g.end;
  }
  a.N = n;
  a.K = (int)s->P;
  a.gy = gy;
  const int tile = wgrad_tile(s, M, n);
  const WgradPlan w = wgrad_plan(s, tile, M, n);
  const int splits = w.splits;
  if ((size_t)w.slots * M * n > s->part_cap)
    return fail(PULSE_E_SHAPE, "internal: wgrad partial buffer too small");
  a.kchunk = w.kchunk;
  a.part = s->sf(s->s_part);
  if (uses_v2(s))
    HIPCHK(launch_wgrad2(a, tile, splits, s->scratch(s->s_zero), st));
  else
    HIPCHK(launch_wgrad(a, tile, splits, st));
  return PULSE_OK;
}

// GroupNorm+SiLU forward of x into dst0/dst1.  pre_chunks > 0: the
// per-chunk channel sums of x are already in the reduction buffer, with that
// many chunks per image (written by the producing conv's epilogue).
// src (null: x) is what the statistics pass reads, and copy (null: none)
// receives its first source as read: the stage's input arrives in the
// caller's buffer and is kept, by the statistics pass, in the row that x
// then points at.
pulse_status gn_forward(pulse_stage* s, char* row, const GnSave& g, const VIn& x,
                        const float* gamma, const float* beta, void* dst0, void* dst1,
                        hipStream_t st, int pre_chunks = 0, const VIn* src = nullptr,
                        void* copy = nullptr) {
  RedGrid rg = red_grid(s->geo, x.C);
  float* red = s->fwd(s->f_red);
  if (pre_chunks > 0)
    rg.chunks = pre_chunks;
  else
    HIPCHK(launch_gn_stats_partial(src ? *src : x, s->geo, rg, red, st, copy));
  float* mean = reinterpret_cast<float*>(row + g.mean);
  float* rstd = reinterpret_cast<float*>(row + g.rstd);
  float* scale = reinterpret_cast<float*>(row + g.scale);
  float* shift = reinterpret_cast<float*>(row + g.shift);
  HIPCHK(launch_gn_stats_finalize(red, s->geo, rg, x.C, s->G, s->eps, gamma, beta, mean, rstd,
                                  scale, shift, st));
  HIPCHK(launch_gn_apply(x, s->geo, scale, shift, dst0, dst1, s->dtype, st));
  return PULSE_OK;
}

// GroupNorm+SiLU backward: da (fp32 [P][C]) -> o (split store + addends)
// pre_chunks > 0: the per-chunk sums are already in the reduction buffer
// (written by the data-gradient conv's epilogue, that many chunks per image).
pulse_status gn_backward(pulse_stage* s, char* row, const GnSave& g, const VIn& x,
                         const float* gamma, float* dgamma, float* dbeta, const void* da_ptr,
                         const GnBwdOut& o, hipStream_t st, int pre_chunks = 0,
                         hipEvent_t done = nullptr) {
  RedGrid rg = red_grid(s->geo, x.C);
  float* red = s->sf(s->s_red);
  float* coef = s->sf(s->s_coef);
  const Src da = src_of(da_ptr, s->dtype, x.C);
  const float* mean = reinterpret_cast<const float*>(row + g.mean);
  const float* rstd = reinterpret_cast<const float*>(row + g.rstd);
  const float* scale = reinterpret_cast<const float*>(row + g.scale);
  const float* shift = reinterpret_cast<const float*>(row + g.shift);
  if (pre_chunks > 0) {
    rg.chunks = pre_chunks;
  } else {
    HIPCHK(launch_gn_bwd_partial(da, x, s->geo, rg, scale, shift, mean, rstd, s->G, red, st));
  }
  HIPCHK(launch_gn_bwd_finalize(red, s->geo, rg, x.C, s->G, gamma, coef, dgamma, dbeta, st));
  // the apply's block grid is its own
  const RedGrid ra = red_grid(s->geo, x.C);
  HIPCHK(launch_gn_bwd_apply(da, x, s->geo, ra, scale, shift, mean, rstd, gamma, coef, s->G, o,
                             st, done));
  return PULSE_OK;
}

// The virtual input (block input) of block b for row `row`.
VIn block_input(pulse_stage* s, int r, const Block& b, int k, const void* dec_up) {
  char* row = s->row_base(r);
  const int dt = s->dtype;
  if (!b.dec) {
    const void* p;
    if (k == 0) {
      p = s->d.input_skip_slot >= 0 ? row + s->row_act[s->d.input_skip_slot] : row + s->row_xin;
    } else {
      const Block& prev = s->eb[k - 1];
      p = prev.slot >= 0 ? row + s->row_act[prev.slot] : row + prev.out_saved;
    }
    return vin1(p, dt, b.cin);
  }
  const void* up = dec_up;
  if (!up) up = (k == 0) ? row + s->row_u : row + s->db[k - 1].out_saved;
  return vin2(up, dt, b.c0, row + s->row_act[b.slot], dt, b.cin - b.c0);
}

// The side stream is used unless per-kernel timing is on: timed conv
// launches then run alone on the caller's stream, so their events measure
// the kernel and not its overlap with the weight-gradient GEMMs.
bool use_side(const pulse_stage* s) { return s->side && !s->timing; }

float* temb_slice(pulse_stage* s, int k) {
  return s->fwd(s->f_e) + (size_t)k * s->geo.B * s->cmax;
}

// One ResBlock forward.  `out` receives the block output, `out2` a copy.
// in_chunks > 0: the GN1 statistics of xin are
// already in the reduction buffer (from the previous block's conv2);
// out_chunks non-null: ask conv2 for the statistics of `out` (receives their
// chunks per image, 0 when not computed).
pulse_status block_forward(pulse_stage* s, int r, const Block& b, const VIn& xin, void* out,
                           void* out2, const float* e, int in_chunks, int* out_chunks,
                           hipStream_t st, const VIn* xsrc = nullptr, void* xcopy = nullptr) {
  char* row = s->row_base(r);
  const int dt = s->dtype;
  void* a1_0 = row + b.a1_0;
  void* a1_1 = row + b.a1_1;
  pulse_status ps;
  // a1 = SiLU(GN1(x)), one tensor per source (the first block's statistics
  // pass reads the caller's input xsrc and keeps it in xin's row buffer)
  if ((ps = gn_forward(s, row, b.gn1, xin, s->pp(b.g1), s->pp(b.be1), a1_0, a1_1, st,
                       in_chunks, xsrc, xcopy)) != PULSE_OK)
    return ps;
  // e = b1 + bl + Wl SiLU(temb), computed for every block of the half
  // beforehand (temb_project)
  const VIn a1 = (b.cin > b.c0) ? vin2(a1_0, dt, b.c0, a1_1, dt, b.cin - b.c0)
                                : vin1(a1_0, dt, b.cin);
  void* h1 = row + b.h1;
  int h1_chunks = 0;  // GN2 statistics of h1 from conv1's epilogue, when it can
  if ((ps = conv_fwd(s, b.cout, {seg3(0, b.cin, a1)}, s->ws + b.wf1, 9 * b.cin, nullptr, e,
                     vnone(), h1, nullptr, dt, st, s->fwd(s->f_red), &h1_chunks)) != PULSE_OK)
    return ps;
  // a2 = SiLU(GN2(h1))
  const VIn h1v = vin1(h1, dt, b.cout);
  void* a2 = row + b.a2;
  if ((ps = gn_forward(s, row, b.gn2, h1v, s->pp(b.g2), s->pp(b.be2), a2, nullptr, st,
                       h1_chunks)) != PULSE_OK)
    return ps;
  const VIn a2v = vin1(a2, dt, b.cout);
  const float* bias2 = reinterpret_cast<const float*>(s->ws + b.bias2);
  float* ostats = out_chunks ? s->fwd(s->f_red) : nullptr;  // GN2 has consumed it
  if (b.conv_sc)
    return conv_fwd(s, b.cout, {seg3(0, b.cout, a2v), seg1(9 * b.cout, b.cin, xin)},
                    s->ws + b.wf2, b.ldb2, bias2, nullptr, vnone(), out, out2, dt, st, ostats,
                    out_chunks);
  return conv_fwd(s, b.cout, {seg3(0, b.cout, a2v)}, s->ws + b.wf2, b.ldb2, bias2, nullptr, xin,
                  out, out2, dt, st, ostats, out_chunks);
}

// One ResBlock backward.  dout: gradient w.r.t. the block output.  o: where

// Fork: work enqueued on the side stream after this starts once everything
// enqueued on `st` so far has finished.  Join: `st` continues once the side
// stream's work so far has finished.  Without a side stream both are no-ops
// and the side work runs on `st`.
pulse_status fork_side(pulse_stage* s, hipStream_t st) {
  if (!use_side(s)) return PULSE_OK;
  // a marker between two kernels costs the stream a few microseconds; an
  // event attached to the producing kernel's completion does not
  if (!s->fork_attached) HIPCHK(hipEventRecord(s->ev_fork, st));
  s->fork_attached = false;
  HIPCHK(hipStreamWaitEvent(s->side, s->ev_fork, 0));
  return PULSE_OK;
}

// The event the next fork may use when the kernel about to be enqueued on
// the caller's stream is the last one before that fork.  Not under stream
// capture: a graph takes its dependencies from recorded events.
hipEvent_t attach_fork(pulse_stage* s, bool fork_follows, hipStream_t st) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (fork_follows && use_side(s) && hipStreamIsCapturing(st, &cs) != hipSuccess)
    cs = hipStreamCaptureStatusActive;  // unknown: take the marker
  s->fork_attached = fork_follows && use_side(s) && cs == hipStreamCaptureStatusNone;
  return s->fork_attached ? s->ev_fork : nullptr;
}

pulse_status mark_side(pulse_stage* s, hipEvent_t ev) {
  if (!use_side(s)) return PULSE_OK;
  HIPCHK(hipEventRecord(ev, s->side));
  return PULSE_OK;
}

pulse_status wait_mark(pulse_stage* s, hipEvent_t ev, bool recorded, hipStream_t st) {
  if (!use_side(s) || !recorded) return PULSE_OK;
  HIPCHK(hipStreamWaitEvent(st, ev, 0));
  return PULSE_OK;
}

// A decoder backward left running beside its stream: `st` waits for all of
// the side stream's work so far.
pulse_status settle_pending(pulse_stage* s, hipStream_t st) {
  if (!s->join_pending) return PULSE_OK;
  HIPCHK(hipEventRecord(s->ev_join, s->side));
  HIPCHK(hipStreamWaitEvent(st, s->ev_join, 0));
  s->join_pending = false;
  return PULSE_OK;
}

// Calls may alternate streams: order this call's work after the previous
// call's (a no-op on the same stream), including side-stream work that a
// decoder backward left running.
pulse_status order_after_last(pulse_stage* s, hipStream_t st) {
  pulse_status ps;
  if ((ps = settle_pending(s, st)) != PULSE_OK) return ps;
  if (s->have_last && s->last_st != st) HIPCHK(hipStreamWaitEvent(st, s->ev_last, 0));
  return PULSE_OK;
}

pulse_status mark_last(pulse_stage* s, hipStream_t st) {
  HIPCHK(hipEventRecord(s->ev_last, st));
  s->last_st = st;
  s->have_last = true;
  return PULSE_OK;
}

pulse_status join_side(pulse_stage* s, hipStream_t st) {
  if (!use_side(s)) return PULSE_OK;
  HIPCHK(hipEventRecord(s->ev_join, s->side));
  HIPCHK(hipStreamWaitEvent(st, s->ev_join, 0));
  return PULSE_OK;
}

// Timestep projections e_k = b1 + bl + Wl SiLU(temb) of every block of one
// half, into consecutive [B][cmax] slices of the e buffer, in one launch per
// 16 blocks on the caller's stream (a side stream would cost an event round
// trip before the first conv); the first launch also keeps temb in the row.
pulse_status temb_project(pulse_stage* s, int r, const std::vector<Block>& blocks, int half,
                          const void* temb, hipStream_t st) {
  char* row = s->row_base(r);
  for (size_t k0 = 0; k0 < blocks.size(); k0 += TEMB_MAX_BLOCKS) {
    TembFwdSet set{};
    set.n = (int)std::min<size_t>(TEMB_MAX_BLOCKS, blocks.size() - k0);
    for (int j = 0; j < set.n; ++j) {
      const Block& b = blocks[k0 + j];
      set.blk[j] = TembFwdBlock{s->pp(b.Wl), s->pp(b.b1), s->pp(b.bl),
                                temb_slice(s, (int)(k0 + j)), b.cout, b.cout};
    }
    HIPCHK(launch_temb_fwd_multi(temb, s->dtype, s->geo.B, s->D, set,
                                 k0 == 0 ? row + s->row_temb[half] : nullptr, st));
  }
  return PULSE_OK;
}

// the gradient w.r.t. the block input goes (split/addends set by caller;
// the residual / shortcut addend is filled in here).  prev_dout: the
// gradient buffer the block processed before this one read as its dout
// (the side stream may still be reading it).
pulse_status block_backward(pulse_stage* s, int r, const Block& b, const VIn& xin,
                            const VIn& dout, GnBwdOut o, float* dtemb, hipStream_t st, int k,
                            BwdSync& sy, const void* prev_dout) {
  const int par = k & 1;
  char* row = s->row_base(r);
  const int dt = s->dtype;
  pulse_status ps;
  // Parameter gradients of conv2 / the shortcut (bias sums and the weight
  // GEMM) only read dout and saved activations: they run on the side stream
  // while the data-gradient chain continues here.  The side stream has its
  // own reduction buffer and weight-gradient partials.
  hipStream_t sd = use_side(s) ? s->side : st;
  // The shortcut's data gradient (a 1x1 conv over dout: short K, its output
  // twice dout's width) runs first and alone when this stage's convs fill
  // the GPU without a K split: beside the weight GEMMs, whose blocks leave no
  // room for its own on their CUs, it took three times as long.  Where the
  // convs split K the weight GEMMs bound the backward, and it stays beside
  // them, after the fork.
  void* dxs = s->scratch(s->s_dxs);
  auto shortcut_dgrad = [&]() -> pulse_status {
    return conv_fwd(s, b.cin, {seg1(0, b.cout, dout)}, s->ws + b.wsd, b.cout, nullptr, nullptr,
                    vnone(), dxs, nullptr, dt, st);
  };
  const bool sc_first =
      b.conv_sc && conv_ksplit(s, conv_tile(s, b.cout), b.cout, 9 * b.cout) == 1;
  if (sc_first) {
    if ((ps = shortcut_dgrad()) != PULSE_OK) return ps;
    s->fork_attached = false;  // the fork below orders the side stream after it
  }
  if ((ps = fork_side(s, st)) != PULSE_OK) return ps;
  {
    const RedGrid rg = red_grid(s->geo, b.cout);
    float* red = s->sf(use_side(s) ? s->s_red2 : s->s_red);
    HIPCHK(launch_chan_sum_partial(dout, s->geo, rg, red, sd));
    HIPCHK(launch_chan_totals(red, s->geo, rg, b.cout, 1, s->gp(b.b2),
                              b.conv_sc ? s->gp(b.bs) : nullptr, nullptr, sd));
  }
  const VIn a2v = vin1(row + b.a2, dt, b.cout);
  if (b.conv_sc) {
    if ((ps = wgrad(s, b.cout,
                    {seg3(0, b.cout, a2v, s->gp(b.W2)), seg1(9 * b.cout, b.cin, xin, s->gp(b.Ws))},
                    dout, sd)) != PULSE_OK)
      return ps;
  } else {
    if ((ps = wgrad(s, b.cout, {seg3(0, b.cout, a2v, s->gp(b.W2))}, dout, sd)) != PULSE_OK)
      return ps;
  }
  if ((ps = mark_side(s, s->ev_w2[par])) != PULSE_OK) return ps;
  sy.w2[par] = true;
  // data gradients through conv2 and the shortcut
  // data gradients are stored in the stage dtype (the MFMA operands they feed
  // are rounded to it anyway; the GroupNorm backward reads them once more)
  void* da = s->scratch(s->s_da);
  // the GroupNorm-backward sums of GN2 (input h1) come from this conv's
  // epilogue when it can produce them (gn2_chunks > 0)
  float* red = s->sf(s->s_red);
  const VIn h1v = vin1(row + b.h1, dt, b.cout);
  const GnbReq gnb2{red, h1v, reinterpret_cast<const float*>(row + b.gn2.scale),
                    reinterpret_cast<const float*>(row + b.gn2.shift),
                    reinterpret_cast<const float*>(row + b.gn2.mean),
                    reinterpret_cast<const float*>(row + b.gn2.rstd)};
  int gn2_chunks = 0;
  if ((ps = conv_fwd(s, b.cout, {seg3(0, b.cout, dout)}, s->ws + b.wd2, 9 * b.cout, nullptr,
                     nullptr, vnone(), da, nullptr, dt, st, nullptr, &gn2_chunks, &gnb2)) !=
      PULSE_OK)
    return ps;
  if (b.conv_sc && !sc_first)
    if ((ps = shortcut_dgrad()) != PULSE_OK) return ps;
  // GN2 backward -> dh1, with per-image channel sums (the temb gradient);
  // dh1 alternates between two buffers: the one written here was last read
  // by the conv1 weight gradient of the block before the previous one
  void* dh1 = s->scratch(s->s_dh1[par]);
  if ((ps = wait_mark(s, s->ev_w1[par], sy.w1[par], st)) != PULSE_OK) return ps;
  {
    GnBwdOut o2{};
    o2.dst0 = dh1;
    o2.dtype0 = dt;
    o2.c_split = b.cout;
    o2.add0 = vnone();
    o2.chan_partial = s->sf(s->s_chp[par]);
    if ((ps = gn_backward(s, row, b.gn2, h1v, s->pp(b.g2), s->gp(b.g2), s->gp(b.be2), da, o2,
                          st, gn2_chunks, attach_fork(s, true, st))) != PULSE_OK)
      return ps;
  }
  // conv1 weight and data gradients
  const VIn a1 = (b.cin > b.c0) ? vin2(row + b.a1_0, dt, b.c0, row + b.a1_1, dt, b.cin - b.c0)
                                : vin1(row + b.a1_0, dt, b.cin);
  const VIn dh1v = vin1(dh1, dt, b.cout);
  if ((ps = fork_side(s, st)) != PULSE_OK) return ps;  // dh1 and its sums are complete
  {
    // the timestep-embedding gradient from the per-image sums of dh1, on the
    // side stream (the next write of this parity's sums waits for ev_w1)
    const RedGrid rg = red_grid(s->geo, b.cout);
    float* de = s->sf(s->s_pi);  // [B][cout]
    HIPCHK(launch_chan_per_image(s->sf(s->s_chp[par]), s->geo, rg, b.cout, 1, de, sd));
    HIPCHK(launch_temb_bwd(de, row + s->row_temb[b.dec ? 1 : 0], dt, s->geo.B, s->D, b.cout,
                           s->pp(b.Wl), s->gp(b.Wl), s->gp(b.bl), s->gp(b.b1), dtemb, sd));
  }
  if ((ps = wgrad(s, b.cout, {seg3(0, b.cin, a1, s->gp(b.W1))}, dh1v, sd)) != PULSE_OK)
    return ps;
  if ((ps = mark_side(s, s->ev_w1[par])) != PULSE_OK) return ps;
  sy.w1[par] = true;
  const GnbReq gnb1{red, xin, reinterpret_cast<const float*>(row + b.gn1.scale),
                    reinterpret_cast<const float*>(row + b.gn1.shift),
                    reinterpret_cast<const float*>(row + b.gn1.mean),
                    reinterpret_cast<const float*>(row + b.gn1.rstd)};
  int gn1_chunks = 0;
  if ((ps = conv_fwd(s, b.cin, {seg3(0, b.cout, dh1v)}, s->ws + b.wd1, 9 * b.cout, nullptr,
                     nullptr, vnone(), da, nullptr, dt, st, nullptr, &gn1_chunks, &gnb1)) !=
      PULSE_OK)
    return ps;
  // GN1 backward + residual path -> gradient w.r.t. the block input
  o.add0 = b.conv_sc ? vin1(dxs, dt, b.cin) : dout;
  o.chan_partial = nullptr;
  // when the GN1 backward writes the gradient buffer that was the previous
  // block's dout, the side stream must have read it (each wait costs this
  // stream an event round trip)
  if (prev_dout && o.dst0 == prev_dout)
    if ((ps = wait_mark(s, s->ev_w2[par ^ 1], sy.w2[par ^ 1], st)) != PULSE_OK) return ps;
  // the next block of this call forks right after this kernel
  return gn_backward(s, row, b.gn1, xin, s->pp(b.g1), s->gp(b.g1), s->gp(b.be1), da, o, st,
                     gn1_chunks, attach_fork(s, k > 0, st));
}

pulse_status check_ptr(const void* p, const char* what) {
  if (!p) return fail(PULSE_E_INVALID_ARG, "%s is NULL", what);
  if (reinterpret_cast<uintptr_t>(p) % 16)
    return fail(PULSE_E_INVALID_ARG, "%s is not 16-byte aligned", what);
  return PULSE_OK;
}

pulse_status need_bound(const pulse_stage* s) {
  if (s->dry) return PULSE_OK;
  if (!s->bound) return fail(PULSE_E_NOT_BOUND, "stage has no bound parameters/workspace");
  if (!s->synced) return fail(PULSE_E_NOT_BOUND, "pulse_stage_sync_params has not run");
  return PULSE_OK;
}

double block_flops(const pulse_stage* s, const Block& b) {
  const double P = (double)s->P;
  double f = 2.0 * P * b.cout * 9 * b.cin + 2.0 * P * b.cout * 9 * b.cout +
             2.0 * s->geo.B * b.cout * s->D;
  if (b.conv_sc) f += 2.0 * P * b.cout * b.cin;
  return f;
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================

namespace {

// The forward pass's scratch for pulse_stage_forward_static: one array per
// GPU, held until the process ends.  Host code never uses its name as an
// address: fwd_scratch_ptr[device] holds the device address, taken with
// hipGetSymbolAddress on the call's device the first time that device is
// used.
constexpr size_t FWD_SCRATCH_BYTES = (size_t)PULSE_FWD_STATIC_SCRATCH_BYTES;
static __device__ __align__(256) char fwd_scratch[FWD_SCRATCH_BYTES];
constexpr int MAX_DEVICES = 64;
std::mutex fwd_scratch_mu;
void* fwd_scratch_ptr[MAX_DEVICES] = {};

pulse_status fwd_scratch_of_current_device(char** out) {
  int dev = -1;
  HIPCHK(hipGetDevice(&dev));
  if (dev < 0 || dev >= MAX_DEVICES) return fail(PULSE_E_INVALID_ARG, "device %d out of range", dev);
  std::lock_guard<std::mutex> lock(fwd_scratch_mu);
  if (!fwd_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(fwd_scratch));
    if (e != hipSuccess || !p)
      return fail(PULSE_E_HIP, "hipGetSymbolAddress of the forward scratch: %s",
                  hipGetErrorString(e));
    fwd_scratch_ptr[dev] = p;
  }
  *out = static_cast<char*>(fwd_scratch_ptr[dev]);
  return PULSE_OK;
}

pulse_status forward_impl(pulse_stage* s, pulse_half half, int32_t mb, const void* in,
                          const void* temb, void* out, void* stream, bool static_scratch) {
  if (!s) return fail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (half != PULSE_ENC && half != PULSE_DEC) return fail(PULSE_E_INVALID_ARG, "bad half");
  if (mb < 0) return fail(PULSE_E_INVALID_ARG, "mb must be >= 0");
  pulse_status ps;
  char* sbase = nullptr;
  if (static_scratch && s->fs_bytes > FWD_SCRATCH_BYTES)
    return fail(PULSE_E_SHAPE,
                "the forward pass of this stage needs %zu bytes of scratch, more than the %zu "
                "of the static array",
                s->fs_bytes, FWD_SCRATCH_BYTES);
  if (!s->dry) {
    if ((ps = need_bound(s)) != PULSE_OK) return ps;
    if ((ps = check_ptr(in, "in")) != PULSE_OK || (ps = check_ptr(temb, "temb")) != PULSE_OK ||
        (ps = check_ptr(out, "out")) != PULSE_OK)
      return ps;
    if (static_scratch) {
      if (s->timing)
        return fail(PULSE_E_STATE, "per-launch timing creates events: switch it off first");
      if ((ps = fwd_scratch_of_current_device(&sbase)) != PULSE_OK) return ps;
    }
  }
  int r = find_row(s, mb);
  const pulse_stage_desc& d = s->d;
  if (half == PULSE_ENC) {
    if (r >= 0 && s->rows[r].state != R_FRESH)
      return fail(PULSE_E_STATE, "mb %d: encoder forward already ran", mb);
    if (r >= 0) {
      const Row& row = s->rows[r];
      if (d.input_skip_slot >= 0 && row.act[d.input_skip_slot])
        return fail(PULSE_E_CACHE_OCCUPIED, "mb %d slot %d already present", mb,
                    d.input_skip_slot);
      for (auto& b : s->eb)
        if (b.slot >= 0 && row.act[b.slot])
          return fail(PULSE_E_CACHE_OCCUPIED, "mb %d slot %d already present", mb, b.slot);
    } else {
      r = free_row(s);
      if (r < 0)
        return fail(PULSE_E_CACHE_FULL, "mb %d: %d microbatches already in flight", mb,
                    d.max_inflight);
    }
  } else {
    if (r < 0) return fail(PULSE_E_STATE, "mb %d: decoder forward before encoder forward", mb);
    const Row& row = s->rows[r];
    if (row.state != R_ENC_FWD && row.state != R_FRESH)
      return fail(PULSE_E_STATE, "mb %d: decoder forward out of order (state %d)", mb, row.state);
    for (auto& b : s->db)
      if (!row.act[b.slot])
        return fail(PULSE_E_CACHE_MISS, "mb %d: skip slot %d absent", mb, b.slot);
  }

  if (!s->dry) {
    hipStream_t st = static_cast<hipStream_t>(stream);
    char* row = s->row_base(r);
    const int dt = s->dtype;
    if (static_scratch) {
      s->fwd_base = sbase;
      s->f_red = s->fs_red;
      s->f_e = s->fs_e;
      s->f_kpart = s->fs_kpart;
      s->f_kcap = s->fs_kcap;
    } else {
      s->use_workspace_scratch();
    }
    if ((ps = order_after_last(s, st)) != PULSE_OK) return ps;
    // the timestep projections of every block of the half (temb kept in the row)
    if ((ps = temb_project(s, r, half == PULSE_ENC ? s->eb : s->db, half == PULSE_DEC ? 1 : 0,
                           temb, st)) != PULSE_OK)
      return ps;
    if (half == PULSE_ENC) {
      // the first statistics pass reads `in` and keeps it where the block
      // input lives (its own row buffer, or the skip slot it also fills)
      void* xin_store = d.input_skip_slot >= 0 ? row + s->row_act[d.input_skip_slot]
                                               : row + s->row_xin;
      const VIn xsrc = vin1(in, dt, s->eb[0].cin);
      const int n = (int)s->eb.size();
      int chunks = 0;  // GN1 statistics of the next block's input, from conv2
      for (int k = 0; k < n; ++k) {
        const Block& b = s->eb[k];
        const VIn xin = block_input(s, r, b, k, nullptr);
        void* o1;
        void* o2 = nullptr;
        if (b.slot >= 0) {
          o1 = row + s->row_act[b.slot];
          if (k == n - 1) o2 = out;
        } else {
          o1 = (k == n - 1) ? out : row + b.out_saved;
        }
        // the next encoder block normalises exactly this output
        const int in_chunks = chunks;
        if ((ps = block_forward(s, r, b, xin, o1, o2, temb_slice(s, k), in_chunks,
                                k + 1 < n ? &chunks : nullptr, st, k == 0 ? &xsrc : nullptr,
                                k == 0 ? xin_store : nullptr)) != PULSE_OK)
          return ps;
      }
    } else {
      const int n = (int)s->db.size();
      for (int k = 0; k < n; ++k) {
        const Block& b = s->db[k];
        const VIn xin = block_input(s, r, b, k, nullptr);
        // block 0 reads u from the caller and keeps it in the row
        VIn xsrc = xin;
        xsrc.s0.ptr = in;
        void* o1 = (k == n - 1) ? out : row + b.out_saved;
        if ((ps = block_forward(s, r, b, xin, o1, nullptr, temb_slice(s, k), 0, nullptr, st,
                                k == 0 ? &xsrc : nullptr,
                                k == 0 ? row + s->row_u : nullptr)) != PULSE_OK)
          return ps;
      }
    }
    if ((ps = mark_last(s, st)) != PULSE_OK) return ps;
  }

  Row& row = s->rows[r];
  if (half == PULSE_ENC) {
    row.mb = mb;
    row.state = R_ENC_FWD;
    row.enc_done = true;
    if (d.input_skip_slot >= 0) row.act[d.input_skip_slot] = 1;
    for (auto& b : s->eb)
      if (b.slot >= 0) row.act[b.slot] = 1;
  } else {
    row.state = R_DEC_FWD;
  }
  return PULSE_OK;
}

}  // namespace

extern "C" {

const char* pulse_last_error(void) { return g_err.c_str(); }

pulse_status pulse_stage_create(const pulse_stage_desc* desc, pulse_stage** out) {
  if (!out) return fail(PULSE_E_INVALID_ARG, "out is NULL");
  *out = nullptr;
  pulse_status st = validate_desc(desc);
  if (st != PULSE_OK) return st;
  pulse_stage* s = new (std::nothrow) pulse_stage();
  if (!s) return fail(PULSE_E_INVALID_ARG, "out of host memory");
  s->d = *desc;
  s->enc.assign(desc->enc, desc->enc + desc->n_enc);
  s->dec.assign(desc->dec, desc->dec + desc->n_dec);
  s->d.enc = s->enc.data();
  s->d.dec = s->dec.data();
  s->dry = (desc->flags & PULSE_FLAG_DRY_RUN) != 0;
  if ((st = build_slots(s)) != PULSE_OK || (st = build_layout(s)) != PULSE_OK) {
    delete s;
    return st;
  }
  s->rows.resize(desc->max_inflight);
  *out = s;
  return PULSE_OK;
}

void pulse_stage_destroy(pulse_stage* s) {
  if (!s) return;
  // work a decoder backward left on the side stream ends before its events go
  if (s->side) (void)hipStreamSynchronize(s->side);
  for (hipEvent_t e : s->ev_pool) (void)hipEventDestroy(e);
  if (s->ev_fork) (void)hipEventDestroy(s->ev_fork);
  if (s->ev_join) (void)hipEventDestroy(s->ev_join);
  for (int i = 0; i < 2; ++i) {
    if (s->ev_w2[i]) (void)hipEventDestroy(s->ev_w2[i]);
    if (s->ev_w1[i]) (void)hipEventDestroy(s->ev_w1[i]);
  }
  if (s->ev_last) (void)hipEventDestroy(s->ev_last);
  if (s->side) (void)hipStreamDestroy(s->side);
  delete s;
}

pulse_status pulse_stage_sizes(const pulse_stage* s, int64_t* n_params, size_t* ws_bytes) {
  if (!s) return fail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (n_params) *n_params = s->n_params;
  if (ws_bytes) *ws_bytes = s->dry ? 0 : s->ws_bytes;
  return PULSE_OK;
}

pulse_status pulse_stage_param_layout(const pulse_stage* s, int32_t idx, char name[64],
                                      int64_t* offset, int32_t shape[4]) {
  if (!s) return fail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (idx == -1) {
    if (!offset) return fail(PULSE_E_INVALID_ARG, "offset is NULL");
    *offset = (int64_t)s->params.size();
    return PULSE_OK;
  }
  if (idx < 0 || idx >= (int)s->params.size())
    return fail(PULSE_E_INVALID_ARG, "parameter index %d out of range", idx);
  const ParamInfo& p = s->params[idx];
  if (name) {
    std::strncpy(name, p.name.c_str(), 63);
    name[63] = 0;
  }
  if (offset) *offset = p.off;
  if (shape)
    for (int i = 0; i < 4; ++i) shape[i] = p.shape[i];
  return PULSE_OK;
}

pulse_status pulse_stage_bind(pulse_stage* s, const float* params, float* grads, void* ws,
                              size_t ws_bytes) {
  if (!s) return fail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (s->dry) return fail(PULSE_E_STATE, "a dry-run stage binds no memory");
  if (!params || !grads || !ws) return fail(PULSE_E_INVALID_ARG, "NULL pointer in bind");
  if (reinterpret_cast<uintptr_t>(ws) % 256 || reinterpret_cast<uintptr_t>(params) % 16 ||
      reinterpret_cast<uintptr_t>(grads) % 16)
    return fail(PULSE_E_INVALID_ARG, "workspace must be 256-byte, params/grads 16-byte aligned");
  if (ws_bytes < s->ws_bytes)
    return fail(PULSE_E_INVALID_ARG, "workspace %zu bytes < required %zu", ws_bytes,
                s->ws_bytes);
  if (pulse_stage_inflight(s) > 0)
    return fail(PULSE_E_STATE, "cannot rebind with microbatches in flight");
  if (!s->ev_last) HIPCHK(hipEventCreateWithFlags(&s->ev_last, hipEventDisableTiming));
  if (!s->side && env_int("PULSE_SERIAL", 0) == 0) {
    // default priority, no implicit synchronisation with the null stream
    HIPCHK(hipStreamCreateWithFlags(&s->side, hipStreamNonBlocking));
    HIPCHK(hipEventCreateWithFlags(&s->ev_fork, hipEventDisableTiming));
    HIPCHK(hipEventCreateWithFlags(&s->ev_join, hipEventDisableTiming));
    for (int i = 0; i < 2; ++i) {
      HIPCHK(hipEventCreateWithFlags(&s->ev_w2[i], hipEventDisableTiming));
      HIPCHK(hipEventCreateWithFlags(&s->ev_w1[i], hipEventDisableTiming));
    }
  }
  s->prm = params;
  s->grd = grads;
  s->ws = static_cast<char*>(ws);
  s->bound = true;
  s->synced = false;
  return PULSE_OK;
}

pulse_status pulse_stage_sync_params(pulse_stage* s, void* stream) {
  if (!s) return fail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (s->dry) {
    s->synced = true;
    return PULSE_OK;
  }
  if (!s->bound) return fail(PULSE_E_NOT_BOUND, "stage is not bound");
  hipStream_t st = static_cast<hipStream_t>(stream);
  pulse_status ps;
  if ((ps = order_after_last(s, st)) != PULSE_OK) return ps;
  const int dt = s->dtype;
  for (auto* v : {&s->eb, &s->db})
    for (auto& b : *v) {
      HIPCHK(launch_convert_rows(s->pp(b.W1), b.cout, 9 * b.cin, s->ws + b.wf1, 9 * b.cin, 0, dt,
                                 st));
      HIPCHK(launch_convert_rows(s->pp(b.W2), b.cout, 9 * b.cout, s->ws + b.wf2, b.ldb2, 0, dt,
                                 st));
      if (b.conv_sc)
        HIPCHK(launch_convert_rows(s->pp(b.Ws), b.cout, b.cin, s->ws + b.wf2, b.ldb2,
                                   9 * b.cout, dt, st));
      HIPCHK(launch_flip3x3(s->pp(b.W1), b.cout, b.cin, s->ws + b.wd1, dt, st));
      HIPCHK(launch_flip3x3(s->pp(b.W2), b.cout, b.cout, s->ws + b.wd2, dt, st));
      if (b.conv_sc) HIPCHK(launch_transpose(s->pp(b.Ws), b.cout, b.cin, s->ws + b.wsd, dt, st));
      HIPCHK(launch_vec_add(s->pp(b.b2), b.conv_sc ? s->pp(b.bs) : nullptr,
                            reinterpret_cast<float*>(s->ws + b.bias2), b.cout, st));
    }
  HIPCHK(hipMemsetAsync(s->scratch(s->s_zero), 0, 256, st));
  if ((ps = mark_last(s, st)) != PULSE_OK) return ps;
  s->synced = true;
  return PULSE_OK;
}

pulse_status pulse_stage_forward(pulse_stage* s, pulse_half half, int32_t mb, const void* in,
                                 const void* temb, void* out, void* stream) {
  return forward_impl(s, half, mb, in, temb, out, stream, false);
}

pulse_status pulse_stage_forward_static(pulse_stage* s, pulse_half half, int32_t mb,
                                        const void* in, const void* temb, void* out,
                                        void* stream) {
  return forward_impl(s, half, mb, in, temb, out, stream, true);
}

pulse_status pulse_stage_backward(pulse_stage* s, pulse_half half, int32_t mb, const void* dout,
                                  void* din, float* dtemb, void* stream) {
  if (!s) return fail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (half != PULSE_ENC && half != PULSE_DEC) return fail(PULSE_E_INVALID_ARG, "bad half");
  if (mb < 0) return fail(PULSE_E_INVALID_ARG, "mb must be >= 0");
  pulse_status ps;
  if (!s->dry) {
    if ((ps = need_bound(s)) != PULSE_OK) return ps;
    if ((ps = check_ptr(dout, "dout")) != PULSE_OK || (ps = check_ptr(din, "din")) != PULSE_OK)
      return ps;
    if (dtemb && reinterpret_cast<uintptr_t>(dtemb) % 4)
      return fail(PULSE_E_INVALID_ARG, "dtemb_accum misaligned");
  }
  const int r = find_row(s, mb);
  if (r < 0) return fail(PULSE_E_STATE, "mb %d is not in flight", mb);
  const pulse_stage_desc& d = s->d;
  {
    const Row& row = s->rows[r];
    if (half == PULSE_DEC && row.state != R_DEC_FWD)
      return fail(PULSE_E_STATE, "mb %d: decoder backward needs the decoder forward", mb);
    if (half == PULSE_ENC) {
      if (row.state != R_DEC_BWD || !row.enc_done)
        return fail(PULSE_E_STATE, "mb %d: encoder backward needs encoder forward and decoder "
                    "backward", mb);
      auto need = [&](int sl) { return sl >= 0 && s->slot_reader[sl] >= 0 && !row.grad[sl]; };
      if (need(d.input_skip_slot))
        return fail(PULSE_E_CACHE_MISS, "mb %d: skip gradient of slot %d absent", mb,
                    d.input_skip_slot);
      for (auto& b : s->eb)
        if (need(b.slot))
          return fail(PULSE_E_CACHE_MISS, "mb %d: skip gradient of slot %d absent", mb, b.slot);
    }
  }

  if (!s->dry) {
    hipStream_t st = static_cast<hipStream_t>(stream);
    char* row = s->row_base(r);
    const int dt = s->dtype;
    s->use_workspace_scratch();
    s->fork_attached = false;
    BwdSync sy;
    if (half == PULSE_ENC && s->join_pending && s->pending_mb == mb && s->pending_st == st &&
        use_side(s)) {
      // The decoder's last parameter-gradient work may still run on the side
      // stream.  Its reads of the blocks' gradient buffers ended at its last
      // conv2 marker, which this stream waits for before writing them; its
      // dh1 and channel-sum buffers are guarded per parity by the carried
      // markers; everything else it reads this call does not write.
      sy = s->sy_pending;
      HIPCHK(hipStreamWaitEvent(st, s->ev_w2[s->par_pending], 0));
      s->join_pending = false;
    } else if ((ps = order_after_last(s, st)) != PULSE_OK) {
      return ps;
    }
    int cur = 0;
    const void* prev_dy = nullptr;  // the dout of the block processed before
    if (half == PULSE_DEC) {
      const int n = (int)s->db.size();
      for (int k = n - 1; k >= 0; --k) {
        const Block& b = s->db[k];
        const VIn xin = block_input(s, r, b, k, nullptr);
        const VIn dy = vin1((k == n - 1) ? dout : s->scratch(s->s_g[cur]), dt, b.cout);
        GnBwdOut o{};
        o.c_split = b.c0;
        o.dst0 = (k == 0) ? din : s->scratch(s->s_g[cur ^ 1]);
        o.dtype0 = dt;
        o.dst1 = row + s->row_grad[b.slot];
        o.dtype1 = DT_F32;
        if ((ps = block_backward(s, r, b, xin, dy, o, dtemb, st, k, sy, prev_dy)) != PULSE_OK)
          return ps;
        prev_dy = dy.s0.ptr;
        cur ^= 1;
      }
    } else {
      const int n = (int)s->eb.size();
      // buffered skip gradient of a slot (null when nothing read the skip)
      auto dskip_of = [&](int slot) -> const float* {
        return (slot >= 0 && s->slot_reader[slot] >= 0)
                   ? reinterpret_cast<const float*>(row + s->row_grad[slot])
                   : nullptr;
      };
      // gradient reaching the last block's output: dout plus its skip gradient
      const void* dlast = dout;
      if (const float* ds = dskip_of(s->eb[n - 1].slot)) {
        HIPCHK(launch_add_cast(dout, dt, ds, s->scratch(s->s_g[cur]), dt,
                               (long)s->P * s->eb[n - 1].cout, st));
        dlast = s->scratch(s->s_g[cur]);
      }
      for (int k = n - 1; k >= 0; --k) {
        const Block& b = s->eb[k];
        const VIn xin = block_input(s, r, b, k, nullptr);
        const VIn dy = vin1((k == n - 1) ? dlast : s->scratch(s->s_g[cur]), dt, b.cout);
        GnBwdOut o{};
        o.c_split = b.cin;
        o.dst0 = (k == 0) ? din : s->scratch(s->s_g[cur ^ 1]);
        o.dtype0 = dt;
        // the block input is the previous block's output (or the stage input):
        // its buffered skip gradient joins here, once
        o.add1 = dskip_of(k == 0 ? d.input_skip_slot : s->eb[k - 1].slot);
        if ((ps = block_backward(s, r, b, xin, dy, o, dtemb, st, k, sy, prev_dy)) != PULSE_OK)
          return ps;
        prev_dy = dy.s0.ptr;
        cur ^= 1;
      }
    }
    if (half == PULSE_DEC && s->overlap_bwd && use_side(s)) {
      // the side stream's remaining work joins at the next call
      s->join_pending = true;
      s->pending_mb = mb;
      s->pending_st = st;
      s->sy_pending = sy;
      s->par_pending = 0;  // the last block processed is block 0
    } else if ((ps = join_side(s, st)) != PULSE_OK) {
      return ps;  // the caller's stream sees every side-stream result
    }
    if ((ps = mark_last(s, st)) != PULSE_OK) return ps;
  }

  Row& row = s->rows[r];
  if (half == PULSE_DEC) {
    row.state = R_DEC_BWD;
    for (auto& b : s->db) row.grad[b.slot] = 1;
  } else {
    release_row(row);
  }
  return PULSE_OK;
}

pulse_status pulse_skip_cache_put(pulse_stage* s, int32_t mb, int32_t slot, const void* src,
                                  void* stream) {
  if (!s) return fail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (mb < 0) return fail(PULSE_E_INVALID_ARG, "mb must be >= 0");
  if (slot < 0 || slot >= s->n_slots || !s->slot_ch[slot])
    return fail(PULSE_E_INVALID_ARG, "slot %d does not exist", slot);
  pulse_status ps;
  if (!s->dry) {
    if (!s->bound) return fail(PULSE_E_NOT_BOUND, "stage is not bound");
    if ((ps = check_ptr(src, "src")) != PULSE_OK) return ps;
  }
  int r = find_row(s, mb);
  if (r >= 0) {
    if (s->rows[r].act[slot])
      return fail(PULSE_E_CACHE_OCCUPIED, "mb %d slot %d already present", mb, slot);
  } else {
    r = free_row(s);
    if (r < 0)
      return fail(PULSE_E_CACHE_FULL, "mb %d: %d microbatches already in flight", mb,
                  s->d.max_inflight);
  }
  if (!s->dry) {
    hipStream_t st = static_cast<hipStream_t>(stream);
    if ((ps = order_after_last(s, st)) != PULSE_OK) return ps;
    HIPCHK(hipMemcpyAsync(s->row_base(r) + s->row_act[slot], src, act_bytes(s, s->slot_ch[slot]),
                          hipMemcpyDeviceToDevice, st));
    if ((ps = mark_last(s, st)) != PULSE_OK) return ps;
  }
  Row& row = s->rows[r];
  if (row.mb < 0) {
    row.mb = mb;
    row.state = R_FRESH;
  }
  row.act[slot] = 1;
  return PULSE_OK;
}

pulse_status pulse_skip_cache_take(pulse_stage* s, int32_t mb, int32_t slot,
                                   pulse_skip_kind kind, void* dst, void* stream) {
  if (!s) return fail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (kind != PULSE_SKIP_ACT && kind != PULSE_SKIP_GRAD)
    return fail(PULSE_E_INVALID_ARG, "bad kind");
  if (slot < 0 || slot >= s->n_slots || !s->slot_ch[slot])
    return fail(PULSE_E_INVALID_ARG, "slot %d does not exist", slot);
  pulse_status ps;
  if (!s->dry) {
    if (!s->bound) return fail(PULSE_E_NOT_BOUND, "stage is not bound");
    if ((ps = check_ptr(dst, "dst")) != PULSE_OK) return ps;
  }
  const int r = find_row(s, mb);
  if (r < 0) return fail(PULSE_E_CACHE_MISS, "mb %d is not in flight", mb);
  Row& row = s->rows[r];
  uint8_t& present = kind == PULSE_SKIP_ACT ? row.act[slot] : row.grad[slot];
  if (!present)
    return fail(PULSE_E_CACHE_MISS, "mb %d slot %d %s absent", mb, slot,
                kind == PULSE_SKIP_ACT ? "activation" : "gradient");
  if (!s->dry) {
    const size_t off = kind == PULSE_SKIP_ACT ? s->row_act[slot] : s->row_grad[slot];
    const size_t bytes = kind == PULSE_SKIP_ACT ? act_bytes(s, s->slot_ch[slot])
                                                : (size_t)s->P * s->slot_ch[slot] * 4;
    hipStream_t st = static_cast<hipStream_t>(stream);
    if ((ps = order_after_last(s, st)) != PULSE_OK) return ps;
    HIPCHK(hipMemcpyAsync(dst, s->row_base(r) + off, bytes, hipMemcpyDeviceToDevice, st));
    if ((ps = mark_last(s, st)) != PULSE_OK) return ps;
  }
  present = 0;
  if (!row.enc_done && (row.state == R_FRESH || row.state == R_DEC_BWD) && row_empty(s, row))
    release_row(row);
  return PULSE_OK;
}

pulse_status pulse_skip_cache_state(const pulse_stage* s, int32_t mb, int32_t slot,
                                    int32_t* state) {
  if (!s || !state) return fail(PULSE_E_INVALID_ARG, "NULL argument");
  if (slot < 0 || slot >= s->n_slots || !s->slot_ch[slot])
    return fail(PULSE_E_INVALID_ARG, "slot %d does not exist", slot);
  const int r = find_row(s, mb);
  *state = 0;
  if (r >= 0)
    *state = (s->rows[r].act[slot] ? PULSE_SKIP_ACT_PRESENT : 0) |
             (s->rows[r].grad[slot] ? PULSE_SKIP_GRAD_PRESENT : 0);
  return PULSE_OK;
}

pulse_status pulse_stage_release(pulse_stage* s, int32_t mb) {
  if (!s) return fail(PULSE_E_INVALID_ARG, "stage is NULL");
  const int r = find_row(s, mb);
  if (r < 0) return fail(PULSE_E_STATE, "mb %d is not in flight", mb);
  release_row(s->rows[r]);
  return PULSE_OK;
}

pulse_status pulse_stage_reset(pulse_stage* s) {
  if (!s) return fail(PULSE_E_INVALID_ARG, "stage is NULL");
  for (auto& r : s->rows) release_row(r);
  return PULSE_OK;
}

int32_t pulse_stage_inflight(const pulse_stage* s) {
  if (!s) return -1;
  int n = 0;
  for (auto& r : s->rows) n += r.mb >= 0;
  return n;
}

pulse_status pulse_stage_overlap_bwd(pulse_stage* s, int32_t enable) {
  if (!s) return fail(PULSE_E_INVALID_ARG, "stage is NULL");
  s->overlap_bwd = enable != 0;
  return PULSE_OK;
}

pulse_status pulse_stage_flush(pulse_stage* s, void* stream) {
  if (!s) return fail(PULSE_E_INVALID_ARG, "stage is NULL");
  if (s->dry) return PULSE_OK;
  return order_after_last(s, static_cast<hipStream_t>(stream));
}

pulse_status pulse_stage_timing(pulse_stage* s, int32_t enable) {
  if (!s) return fail(PULSE_E_INVALID_ARG, "stage is NULL");
  s->timing = enable != 0;
  s->timed.clear();
  s->ev_used = 0;
  return PULSE_OK;
}

pulse_status pulse_stage_timing_read(pulse_stage* s, int64_t* launches, double* ms,
                                     double* flops, double* bytes) {
  if (!s) return fail(PULSE_E_INVALID_ARG, "stage is NULL");
  double t = 0.0, f = 0.0, by = 0.0;
  for (const auto& tl : s->timed) {
    HIPCHK(hipEventSynchronize(tl.b));
    float x = 0.f;
    HIPCHK(hipEventElapsedTime(&x, tl.a, tl.b));
    t += x;
    f += tl.flops;
    by += tl.bytes;
  }
  if (launches) *launches = (int64_t)s->timed.size();
  if (ms) *ms = t;
  if (flops) *flops = f;
  if (bytes) *bytes = by;
  s->timed.clear();
  s->ev_used = 0;
  return PULSE_OK;
}

double pulse_stage_flops(const pulse_stage* s) {
  if (!s) return 0.0;
  double f = 0.0;
  for (auto& b : s->eb) f += block_flops(s, b);
  for (auto& b : s->db) f += block_flops(s, b);
  return 3.0 * f;
}

}  // extern "C"
