// GroupNorm + SiLU forward/backward and per-channel reductions over NHWC
// activations (gfx950).  All of it is HBM-bound streaming: a block owns one
// image, one chunk of pixels and 64 channel vectors of 8 channels; its 256
// threads are 64 channel vectors x 4 pixel lanes, so each pixel row of a
// block is one contiguous, coalesced read.  Reductions are deterministic:
// fixed per-thread order, a fixed LDS tree, per-(image, chunk) partials and
// a finalize that sums them in a fixed order (group sums in fp64).
#include <hip/hip_ext.h>

#include "common.hpp"
#include "kernels.hpp"

namespace pulse {

namespace {

// Block shape of the per-channel kernels: rg.vx channel vectors (8 channels
// each) x rg.py pixel lanes, at most 256 threads; blockIdx.z picks the
// channel-vector slice.
struct Range {
  int b, p0, p1, v, c;
  bool active;
};

__device__ __forceinline__ Range block_range(const Geo& g, RedGrid rg, int C) {
  Range r;
  r.b = blockIdx.x;
  r.p0 = blockIdx.y * rg.cp;
  r.p1 = min(r.p0 + rg.cp, g.hw());
  r.v = blockIdx.z * rg.vx + threadIdx.x;
  r.c = r.v * 8;
  r.active = threadIdx.x < rg.vx && r.c < C;
  return r;
}

// Sum the pixel lanes of NV values per thread through LDS and store the
// block's totals: component i < 8 of channel vector v to row0[8 v + i],
// component 8 + i to row1[8 v + i] (v = this block's channel vectors, those
// below C / 8).  Values go to LDS component-major (conflict-free), and
// every thread of the block then sums some of the vx * NV totals over the
// py lanes in a fixed order.  sm holds NV * 256 floats.
template <int NV>
__device__ __forceinline__ void lane_reduce_store(float (&v)[NV], float* sm, RedGrid rg, int C,
                                                  float* row0, float* row1) {
  const int t = threadIdx.y * rg.vx + threadIdx.x;
  const int nt = rg.vx * rg.py;
#pragma unroll
  for (int i = 0; i < NV; ++i) sm[i * 256 + t] = v[i];
  __syncthreads();
  for (int q = t; q < rg.vx * NV; q += nt) {
    const int i = q / rg.vx, tx = q - i * rg.vx;
    float s = 0.f;
    for (int y = 0; y < rg.py; ++y) s += sm[i * 256 + y * rg.vx + tx];
    const int c = ((int)blockIdx.z * rg.vx + tx) * 8;
    if (c >= C) continue;
    if (i < 8)
      row0[c + i] = s;
    else
      row1[c + i - 8] = s;
  }
}

// ---- per-thread resolved channel vectors ------------------------------------
// Every streaming kernel below gives each thread one vector of 8 channels
// [c, c+8) for all the pixels it visits.  The source tensor of those
// channels (one of a virtual input's two sources), their offset and the
// pixel stride are resolved once, the element type is a template argument,
// and the pixel loop issues all its loads before any use, without branches,
// so that they stay in flight together.

struct Ch8 {
  const void* p;  // tensor base
  long c;         // channel offset inside a pixel
  long stride;    // elements per pixel
};

__device__ __forceinline__ Ch8 resolve(const Src& s, int c) { return Ch8{s.ptr, c, s.C}; }

__device__ __forceinline__ Ch8 resolve(const VIn& v, int c) {
  return c < v.c0 ? Ch8{v.s0.ptr, c, v.s0.C} : Ch8{v.s1.ptr, c - v.c0, v.s1.C};
}

// channels of pixel `pix` as fp32 (DT: element type of the tensor)
template <int DT>
__device__ __forceinline__ void rd8(const Ch8& h, long pix, float v[8]) {
  const long e = pix * h.stride + h.c;
  if constexpr (DT == DT_BF16) {
    const uint4 q = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(h.p) + e);
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  } else {
    const float4* q = reinterpret_cast<const float4*>(static_cast<const float*>(h.p) + e);
    const float4 a = q[0], b = q[1];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
}

// fp32 addend of pixel `pix` (add: tensor base offset by the channel)
__device__ __forceinline__ void add8(const float* add, long stride, long pix, float v[8]) {
  const float4* q = reinterpret_cast<const float4*>(add + pix * stride);
  const float4 a = q[0], b = q[1];
  v[0] += a.x; v[1] += a.y; v[2] += a.z; v[3] += a.w;
  v[4] += b.x; v[5] += b.y; v[6] += b.z; v[7] += b.w;
}

// A thread's view of a virtual input: resolved source plus optional addend.
struct VCh8 {
  Ch8 h;
  const float* add;
  long astride;
};

__device__ __forceinline__ VCh8 resolve_v(const VIn& v, int c) {
  return VCh8{resolve(v, c), v.add ? v.add + c : nullptr, v.C};
}

template <int DT, bool ADD>
__device__ __forceinline__ void rdv8(const VCh8& h, long pix, float v[8]) {
  rd8<DT>(h.h, pix, v);
  if constexpr (ADD) add8(h.add, h.astride, pix, v);
}

// The U pixels p, p + py, ... of one loop step: absolute pixel indices with
// the ones past p1 clamped to the last valid pixel (they are loaded but
// weighted 0), and their weights.
template <int U>
__device__ __forceinline__ void step_pixels(int p, int py, int p1, long img0, long (&pix)[U],
                                            float (&w)[U]) {
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int pu = p + u * py;
    pix[u] = img0 + (pu < p1 ? pu : p1 - 1);
    w[u] = pu < p1 ? 1.f : 0.f;
  }
}

// The backward pass runs the data-gradient chain beside the weight-gradient
// GEMMs of a second stream, whose blocks hold 2 waves of 208 registers on
// every SIMD: kernels of that chain that need at most 96 registers (5 waves
// per SIMD) and 256-thread blocks still find room on those CUs instead of
// waiting for the GEMM to drain.
constexpr int GN_WAVES = 5;
constexpr int U_STATS = 4;  // pixels per loop step of the reductions
constexpr int U_BWD = 1;    // of the backward reductions (within 96 registers)
constexpr int U_APPLY = 1;  // of the backward apply (within 96 registers)

// copy (null: none) receives the channels below x.c0 of every pixel, as
// read ([P][x.c0], the element type of x): the stage keeps its input for the
// backward without a pass of its own.
template <int DT, bool ADD, int U = U_STATS>
__global__ __launch_bounds__(256) void k_gn_stats_partial(VIn x, Geo g, RedGrid rg,
                                                          float* partial, void* copy) {
  __shared__ float sm[256 * 16];
  const Range r = block_range(g, rg, x.C);
  float acc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.f;
  if (r.active) {
    const VCh8 h = resolve_v(x, r.c);
    const long img0 = (long)r.b * g.hw();
    const bool cp = copy && r.c < x.c0;
    for (int p = r.p0 + threadIdx.y; p < r.p1; p += U * rg.py) {
      long pix[U];
      float w[U], f[U][8];
      step_pixels<U>(p, rg.py, r.p1, img0, pix, w);
#pragma unroll
      for (int u = 0; u < U; ++u) rdv8<DT, ADD>(h, pix[u], f[u]);
      if (cp) {
#pragma unroll
        for (int u = 0; u < U; ++u)
          if (p + u * rg.py < r.p1) st8(copy, DT, x.c0, pix[u], r.c, f[u]);
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float v = w[u] * f[u][i];
          acc[i] += v;
          acc[8 + i] += v * f[u][i];
        }
    }
  }
  float* base = partial + ((long)r.b * rg.chunks + blockIdx.y) * 2 * x.C;
  lane_reduce_store<16>(acc, sm, rg, x.C, base, base + x.C);
}

// Fixed-order block sum of two fp64 values (256 threads).
__device__ __forceinline__ void block_sum2(double& a, double& b, double* sm) {
  const int t = threadIdx.x;
  sm[t] = a;
  sm[256 + t] = b;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (t < off) {
      sm[t] += sm[t + off];
      sm[256 + t] += sm[256 + t + off];
    }
    __syncthreads();
  }
  a = sm[0];
  b = sm[256];
}

// one block per (image, group): mean / rstd from the per-chunk channel sums,
// then the folded affine of the group's channels
__global__ __launch_bounds__(256) void k_gn_stats_finalize(const float* partial, Geo g,
                                                           RedGrid rg, int C, int G, float eps,
                                                           const float* gamma, const float* beta,
                                                           float* mean, float* rstd,
                                                           float* scale, float* shift) {
  __shared__ double sm[512];
  const int b = blockIdx.x, gi = blockIdx.y;
  const int cg = C / G;
  double S = 0.0, Q = 0.0;
  // NB loads in flight per thread, added in ascending i
  constexpr int NB = 8;
  const int n = rg.chunks * cg;
  for (int i0 = threadIdx.x; i0 < n; i0 += NB * 256) {
    float s[NB], q[NB];
#pragma unroll
    for (int k = 0; k < NB; ++k) {
      const int i = i0 + k * 256;
      s[k] = q[k] = 0.f;
      if (i < n) {
        const int ch = i / cg;
        const int c = gi * cg + (i - ch * cg);
        const float* base = partial + ((long)b * rg.chunks + ch) * 2 * C;
        s[k] = base[c];
        q[k] = base[C + c];
      }
    }
#pragma unroll
    for (int k = 0; k < NB; ++k)
      if (i0 + k * 256 < n) {
        S += s[k];
        Q += q[k];
      }
  }
  block_sum2(S, Q, sm);
  const double cnt = (double)g.hw() * cg;
  const double m = S / cnt;
  double var = Q / cnt - m * m;
  if (var < 0.0) var = 0.0;
  const float rs = (float)(1.0 / sqrt(var + (double)eps));
  if (threadIdx.x == 0) {
    mean[b * G + gi] = (float)m;
    rstd[b * G + gi] = rs;
  }
  for (int c = gi * cg + threadIdx.x; c < (gi + 1) * cg; c += 256) {
    const float sc = gamma[c] * rs;
    scale[(long)b * C + c] = sc;
    shift[(long)b * C + c] = beta[c] - (float)m * sc;
  }
}

// a = SiLU(x * scale + shift) for the channels of one thread over its
// chunk of pixels; channels below x.c0 go to dst0 (x.c0 channels per pixel),
// the others to dst1 (x.C - x.c0 per pixel).
template <int DT, bool ADD>
__global__ __launch_bounds__(256) void k_gn_apply(VIn x, Geo g, RedGrid rg, const float* scale,
                                                  const float* shift, void* dst0, void* dst1) {
  const Range r = block_range(g, rg, x.C);
  if (!r.active) return;
  const VCh8 h = resolve_v(x, r.c);
  const bool first = r.c < x.c0;
  void* dst = first ? dst0 : dst1;
  const long dstride = first ? x.c0 : x.C - x.c0;
  const long dc = first ? r.c : r.c - x.c0;
  float ss[8], hh[8];
  {
    const float4* sc = reinterpret_cast<const float4*>(scale + (long)r.b * x.C + r.c);
    const float4* sh = reinterpret_cast<const float4*>(shift + (long)r.b * x.C + r.c);
    const float4 s0 = sc[0], s1 = sc[1], h0 = sh[0], h1 = sh[1];
    ss[0] = s0.x; ss[1] = s0.y; ss[2] = s0.z; ss[3] = s0.w;
    ss[4] = s1.x; ss[5] = s1.y; ss[6] = s1.z; ss[7] = s1.w;
    hh[0] = h0.x; hh[1] = h0.y; hh[2] = h0.z; hh[3] = h0.w;
    hh[4] = h1.x; hh[5] = h1.y; hh[6] = h1.z; hh[7] = h1.w;
  }
  const long img0 = (long)r.b * g.hw();
  for (int p = r.p0 + threadIdx.y; p < r.p1; p += U_STATS * rg.py) {
    long pix[U_STATS];
    float w[U_STATS], f[U_STATS][8];
    step_pixels<U_STATS>(p, rg.py, r.p1, img0, pix, w);
#pragma unroll
    for (int u = 0; u < U_STATS; ++u) rdv8<DT, ADD>(h, pix[u], f[u]);
#pragma unroll
    for (int u = 0; u < U_STATS; ++u) {
      if (p + u * rg.py >= r.p1) break;
#pragma unroll
      for (int j = 0; j < 8; ++j) f[u][j] = silu_f(f[u][j] * ss[j] + hh[j]);
      st8(dst, DT, (int)dstride, pix[u], (int)dc, f[u]);
    }
  }
}

// Per-thread constants of the GroupNorm backward for 8 channels of image b.
struct GnConst {
  float sc[8], sh[8], mu[8], rs[8];
};

__device__ __forceinline__ void load8f(const float* p, float v[8]) {
  const float4 a = reinterpret_cast<const float4*>(p)[0];
  const float4 b = reinterpret_cast<const float4*>(p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

// Per-group value of each of the channels [c, c+8) (c a multiple of 8).
// When a group has 4 or at least 8 channels those 8 channels touch at most
// two groups, g0 = c / cg and g1 = (c + 7) / cg, and two loads suffice.
__device__ __forceinline__ void load_group_pair(const float* v, int b, int G, int c, int cg,
                                                float out[8]) {
  if (cg == 4 || cg >= 8) {
    const int g0 = c / cg, g1 = (c + 7) / cg;
    const float a0 = v[b * G + g0], a1 = v[b * G + g1];
#pragma unroll
    for (int j = 0; j < 8; ++j) out[j] = (c + j) / cg == g0 ? a0 : a1;
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) out[j] = v[b * G + (c + j) / cg];
  }
}

__device__ __forceinline__ void load_gn_const(GnConst& k, int b, int c, int C, int G,
                                              const float* scale, const float* shift,
                                              const float* mean, const float* rstd) {
  const int cg = C / G;
  load8f(scale + (long)b * C + c, k.sc);
  load8f(shift + (long)b * C + c, k.sh);
  load_group_pair(mean, b, G, c, cg, k.mu);
  load_group_pair(rstd, b, G, c, cg, k.rs);
}

template <int DT, bool ADD, int U = U_BWD>
__global__ __launch_bounds__(256, GN_WAVES) void k_gn_bwd_partial(Src da, VIn x, Geo g,
                                                        RedGrid rg, const float* scale,
                                                        const float* shift, const float* mean,
                                                        const float* rstd, int G,
                                                        float* partial) {
  __shared__ float sm[256 * 16];
  const Range r = block_range(g, rg, x.C);
  float acc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.f;
  if (r.active) {
    GnConst k;
    load_gn_const(k, r.b, r.c, x.C, G, scale, shift, mean, rstd);
    const VCh8 hx = resolve_v(x, r.c);
    const Ch8 hd = resolve(da, r.c);
    const long img0 = (long)r.b * g.hw();
    for (int p = r.p0 + threadIdx.y; p < r.p1; p += U * rg.py) {
      long pix[U];
      float w[U], f[U][8], d[U][8];
      step_pixels<U>(p, rg.py, r.p1, img0, pix, w);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        rdv8<DT, ADD>(hx, pix[u], f[u]);
        rd8<DT>(hd, pix[u], d[u]);
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float z = f[u][j] * k.sc[j] + k.sh[j];
          const float dz = w[u] * d[u][j] * dsilu_f(z);
          const float xh = (f[u][j] - k.mu[j]) * k.rs[j];
          acc[j] += dz;
          acc[8 + j] += dz * xh;
        }
    }
  }
  float* base = partial + ((long)r.b * rg.chunks + blockIdx.y) * 2 * x.C;
  lane_reduce_store<16>(acc, sm, rg, x.C, base, base + x.C);
}

// Per-image channel sums of the partials: pi[s][b][c] = sum_chunk
// partial[b][chunk][s][c] for the first `nslot` slots.  A block holds 64
// channels x 4 chunk lanes of one image; each lane keeps four loads in
// flight.
constexpr int VX = 64;
constexpr int PY = 4;

__global__ __launch_bounds__(256) void k_chan_per_image(const float* partial, int chunks, int B,
                                                        int C, int nslot, float* pi) {
  __shared__ float sm[2][PY][VX];
  const int c = blockIdx.x * VX + threadIdx.x;
  const int b = blockIdx.y;
  float s0 = 0.f, s1 = 0.f;
  if (c < C) {
    const long stride = 2L * C;
    const float* base = partial + (long)b * chunks * stride + c;
    int ch = threadIdx.y;
    for (; ch + 3 * PY < chunks; ch += 4 * PY) {
      const float a0 = base[(ch + 0 * PY) * stride], a1 = base[(ch + 1 * PY) * stride];
      const float a2 = base[(ch + 2 * PY) * stride], a3 = base[(ch + 3 * PY) * stride];
      s0 += a0;
      s0 += a1;
      s0 += a2;
      s0 += a3;
      if (nslot > 1) {
        const float e0 = base[(ch + 0 * PY) * stride + C], e1 = base[(ch + 1 * PY) * stride + C];
        const float e2 = base[(ch + 2 * PY) * stride + C], e3 = base[(ch + 3 * PY) * stride + C];
        s1 += e0;
        s1 += e1;
        s1 += e2;
        s1 += e3;
      }
    }
    for (; ch < chunks; ch += PY) {
      s0 += base[ch * stride];
      if (nslot > 1) s1 += base[ch * stride + C];
    }
  }
  sm[0][threadIdx.y][threadIdx.x] = s0;
  sm[1][threadIdx.y][threadIdx.x] = s1;
  __syncthreads();
  if (threadIdx.y == 0 && c < C) {
    float t0 = sm[0][0][threadIdx.x], t1 = sm[1][0][threadIdx.x];
#pragma unroll
    for (int y = 1; y < PY; ++y) {
      t0 += sm[0][y][threadIdx.x];
      t1 += sm[1][y][threadIdx.x];
    }
    pi[(long)b * C + c] = t0;
    if (nslot > 1) pi[(long)(B + b) * C + c] = t1;
  }
}

// Channel totals over every image and chunk in one pass: slot 0 is added to
// acc0 (and dup), slot 1 to acc1.  A 256-thread block holds 8 channels x
// 32 row lanes; lane y sums the (image, chunk) rows y, y+32, ... (8 loads
// in flight, added in ascending row order) and the lanes meet in a fixed
// LDS tree.  Small blocks and few registers: the kernel finds room beside
// the GEMMs of the other stream.
constexpr int TX = 8, TY = 32;

__device__ __forceinline__ void chan_totals_block(const float* partial, int rows, int C,
                                                  int nslot, int cblock, float* acc0,
                                                  float* dup, float* acc1,
                                                  float (&sm)[2][TY][TX]) {
  const int tx = threadIdx.x % TX, ty = threadIdx.x / TX;
  const int c = cblock * TX + tx;
  float s0 = 0.f, s1 = 0.f;
  if (c < C) {
    const long stride = 2L * C;
    const float* base = partial + c;
    constexpr int NB = 8;
    for (int i0 = ty; i0 < rows; i0 += NB * TY) {
      float a[NB], e[NB];
#pragma unroll
      for (int k = 0; k < NB; ++k) {
        const int i = i0 + k * TY;
        a[k] = i < rows ? base[(long)i * stride] : 0.f;
        e[k] = (nslot > 1 && i < rows) ? base[(long)i * stride + C] : 0.f;
      }
#pragma unroll
      for (int k = 0; k < NB; ++k)
        if (i0 + k * TY < rows) {
          s0 += a[k];
          s1 += e[k];
        }
    }
  }
  sm[0][ty][tx] = s0;
  sm[1][ty][tx] = s1;
  __syncthreads();
  for (int off = TY / 2; off > 0; off >>= 1) {
    if (ty < off) {
      sm[0][ty][tx] += sm[0][ty + off][tx];
      sm[1][ty][tx] += sm[1][ty + off][tx];
    }
    __syncthreads();
  }
  if (ty == 0 && c < C) {
    if (acc0) acc0[c] += sm[0][0][tx];
    if (dup) dup[c] += sm[0][0][tx];
    if (acc1) acc1[c] += sm[1][0][tx];
  }
}

__global__ __launch_bounds__(256, GN_WAVES) void k_chan_totals(const float* partial, int rows, int C,
                                                     int nslot, float* acc0, float* dup,
                                                     float* acc1) {
  __shared__ float sm[2][TY][TX];
  chan_totals_block(partial, rows, C, nslot, blockIdx.x, acc0, dup, acc1, sm);
}

// GroupNorm backward finalize in one launch of 256-thread blocks: blocks
// [0, B*G) each reduce one (image, group) to coef = (sum gamma*dz,
// sum gamma*dz*xhat) / count in fp64, with every load in flight before the
// sums; blocks [B*G, B*G + ceil(C/8)) add dbeta (sum dz) and dgamma
// (sum dz * xhat) over every image and chunk.
__global__ __launch_bounds__(256, GN_WAVES) void k_gn_bwd_finalize(const float* partial, Geo g,
                                                         RedGrid rg, int C, int G,
                                                         const float* gamma, float* coef,
                                                         float* dgamma, float* dbeta) {
  __shared__ float smc[2][TY][TX];
  __shared__ double sm[512];
  const int nbg = g.B * G;
  if ((int)blockIdx.x >= nbg) {
    chan_totals_block(partial, g.B * rg.chunks, C, 2, blockIdx.x - nbg, dbeta, nullptr, dgamma,
                      smc);
    return;
  }
  const int b = blockIdx.x / G, gi = blockIdx.x - b * G;
  const int cg = C / G;
  double S1 = 0.0, S2 = 0.0;
  constexpr int NB = 8;  // loads in flight per thread, added in ascending i
  const int n = rg.chunks * cg;
  for (int i0 = threadIdx.x; i0 < n; i0 += NB * 256) {
    float ga[NB], p1[NB], p2[NB];
#pragma unroll
    for (int k = 0; k < NB; ++k) {
      const int i = i0 + k * 256;
      ga[k] = p1[k] = p2[k] = 0.f;
      if (i < n) {
        const int ch = i / cg;
        const int c = gi * cg + (i - ch * cg);
        const float* base = partial + ((long)b * rg.chunks + ch) * 2 * C;
        ga[k] = gamma[c];
        p1[k] = base[c];
        p2[k] = base[C + c];
      }
    }
#pragma unroll
    for (int k = 0; k < NB; ++k)
      if (i0 + k * 256 < n) {
        S1 += (double)ga[k] * p1[k];
        S2 += (double)ga[k] * p2[k];
      }
  }
  block_sum2(S1, S2, sm);
  if (threadIdx.x == 0) {
    const double cnt = (double)g.hw() * cg;
    coef[(b * G + gi) * 2 + 0] = (float)(S1 / cnt);
    coef[(b * G + gi) * 2 + 1] = (float)(S2 / cnt);
  }
}

// CHAN: the output's per-chunk channel sums are written (the timestep-
// embedding gradient); ADD0: the addend o.add0 (stage dtype) exists; NF: the
// number of fp32 addends (o.add0's own and o.add1, in that order).  Each
// instance keeps only the registers it needs.
template <int DT, bool CHAN, bool ADD0, int NF, int U = U_APPLY>
__global__ __launch_bounds__(256, GN_WAVES) void k_gn_bwd_apply(Src da, VIn x, Geo g,
                                                      RedGrid rg, const float* scale,
                                                      const float* shift, const float* mean,
                                                      const float* rstd, const float* gamma,
                                                      const float* coef, int G, GnBwdOut o) {
  __shared__ float sm[CHAN ? 256 * 8 : 1];
  const Range r = block_range(g, rg, x.C);
  const int C = x.C;
  const int cg = C / G;
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
  if (r.active) {
    // out = rstd * (gamma * dz - c0 - xhat * c1) with xhat = (x - mean) * rstd,
    // folded per channel into out = A dz + Bq x + Cq (fewer live registers)
    float sc[8], sh[8], A[8], Bq[8], Cq[8];
    {
      GnConst k;
      load_gn_const(k, r.b, r.c, C, G, scale, shift, mean, rstd);
      float ga[8], c0[8], c1[8];
      load8f(gamma + r.c, ga);
      if (cg == 4 || cg >= 8) {  // the 8 channels touch at most two groups
        const int g0 = r.c / cg, g1 = (r.c + 7) / cg;
        const float2 e0 = reinterpret_cast<const float2*>(coef)[r.b * G + g0];
        const float2 e1 = reinterpret_cast<const float2*>(coef)[r.b * G + g1];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const bool first = (r.c + j) / cg == g0;
          c0[j] = first ? e0.x : e1.x;
          c1[j] = first ? e0.y : e1.y;
        }
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float2 e = reinterpret_cast<const float2*>(coef)[r.b * G + (r.c + j) / cg];
          c0[j] = e.x;
          c1[j] = e.y;
        }
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        sc[j] = k.sc[j];
        sh[j] = k.sh[j];
        A[j] = k.rs[j] * ga[j];
        Bq[j] = -k.rs[j] * k.rs[j] * c1[j];
        Cq[j] = -k.rs[j] * c0[j] - Bq[j] * k.mu[j];
      }
    }
    const Ch8 hx = resolve(x, r.c);
    const Ch8 hd = resolve(da, r.c);
    const Ch8 h0 = ADD0 ? resolve(o.add0, r.c) : hx;
    // fp32 addends: o.add0's own first, then o.add1 (both C channels per pixel)
    const bool own = ADD0 && o.add0.add;
    const float* fa0 = own ? o.add0.add + r.c : (o.add1 ? o.add1 + r.c : nullptr);
    const float* fa1 = own && o.add1 ? o.add1 + r.c : nullptr;
    const bool first = r.c < o.c_split;
    void* dst = first ? o.dst0 : o.dst1;
    const int dtype = first ? o.dtype0 : o.dtype1;
    const int dstride = first ? o.c_split : C - o.c_split;
    const int dc = first ? r.c : r.c - o.c_split;
    const long img0 = (long)r.b * g.hw();
    for (int p = r.p0 + threadIdx.y; p < r.p1; p += U * rg.py) {
      long pix[U];
      float w[U], f[U][8], d[U][8], e[U][8];
      step_pixels<U>(p, rg.py, r.p1, img0, pix, w);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        rd8<DT>(hx, pix[u], f[u]);
        rd8<DT>(hd, pix[u], d[u]);
        if constexpr (ADD0) {
          rd8<DT>(h0, pix[u], e[u]);
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j) e[u][j] = 0.f;
        }
        if constexpr (NF >= 1) add8(fa0, C, pix[u], e[u]);
        if constexpr (NF >= 2) add8(fa1, C, pix[u], e[u]);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (p + u * rg.py >= r.p1) break;
        float out[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float dz = d[u][j] * dsilu_f(f[u][j] * sc[j] + sh[j]);
          out[j] = A[j] * dz + (Bq[j] * f[u][j] + Cq[j]) + e[u][j];
        }
        st8(dst, dtype, dstride, pix[u], dc, out);
        if (CHAN) {
#pragma unroll
          for (int j = 0; j < 8; ++j) acc[j] += out[j];
        }
      }
    }
  }
  if (CHAN) {
    float* base = o.chan_partial + ((long)r.b * rg.chunks + blockIdx.y) * 2 * C;
    lane_reduce_store<8>(acc, sm, rg, C, base, nullptr);
  }
}

template <int DT, bool ADD>
__global__ __launch_bounds__(256) void k_chan_sum_partial(VIn v, Geo g, RedGrid rg,
                                                          float* partial) {
  __shared__ float sm[256 * 8];
  const Range r = block_range(g, rg, v.C);
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
  if (r.active) {
    const VCh8 h = resolve_v(v, r.c);
    const long img0 = (long)r.b * g.hw();
    for (int p = r.p0 + threadIdx.y; p < r.p1; p += U_STATS * rg.py) {
      long pix[U_STATS];
      float w[U_STATS], f[U_STATS][8];
      step_pixels<U_STATS>(p, rg.py, r.p1, img0, pix, w);
#pragma unroll
      for (int u = 0; u < U_STATS; ++u) rdv8<DT, ADD>(h, pix[u], f[u]);
#pragma unroll
      for (int u = 0; u < U_STATS; ++u)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] += w[u] * f[u][j];
    }
  }
  float* base = partial + ((long)r.b * rg.chunks + blockIdx.y) * 2 * v.C;
  lane_reduce_store<8>(acc, sm, rg, v.C, base, nullptr);
}

// K-split conv finalize with the statistics of its output, on the grid of
// the GroupNorm kernels: thread (channel vector, pixel lane) sums the fp32
// partials of its 8 channels in split order (two pixels per step, their
// loads in flight together), adds bias, the timestep row and the residual,
// stores bf16 and accumulates the sum and sum of squares of the stored
// values; the lanes meet in LDS (one row per chunk).  (The GroupNorm-
// backward sums measured slower here than in their own pass.)
__global__ __launch_bounds__(256) void k_splitk_finalize_stats(GemmArgs a, RedGrid rg) {
  __shared__ float sm[256 * 16];
  const Geo g = a.g;
  const int N = a.N;
  const Range r = block_range(g, rg, N);
  float acc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.f;
  if (r.active) {
    const long zs = g.pixels() * (long)N;
    float cb[8], cr[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) cb[q] = cr[q] = 0.f;
    if (a.bias) load8f(a.bias + r.c, cb);
    if (a.rowvec) load8f(a.rowvec + (long)r.b * N + r.c, cr);
    const long img0 = (long)r.b * g.hw();
    constexpr int U = 2;
    for (int p = r.p0 + threadIdx.y; p < r.p1; p += U * rg.py) {
      long px[U];
      float w[U];
      step_pixels<U>(p, rg.py, r.p1, img0, px, w);
      float vv[U][8];
#pragma unroll
      for (int u = 0; u < U; ++u) load8f(a.part + px[u] * N + r.c, vv[u]);
      for (int zz = 1; zz < a.ksplit; ++zz) {
        float t[U][8];
#pragma unroll
        for (int u = 0; u < U; ++u) load8f(a.part + zz * zs + px[u] * N + r.c, t[u]);
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
          for (int q = 0; q < 8; ++q) vv[u][q] += t[u][q];
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (p + u * rg.py >= r.p1) break;
        float* v = vv[u];
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] += cb[q];
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] += cr[q];
        if (a.resid.s0.ptr) {
          float t[8];
          ld8(a.resid.s0, px[u], r.c, t);
#pragma unroll
          for (int q = 0; q < 8; ++q) v[q] += t[q];
        }
        st8(a.out, DT_BF16, a.ldo, px[u], r.c, v);
        if (a.out2) st8(a.out2, DT_BF16, a.ldo, px[u], r.c, v);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const float b = bf2f(f2bf(v[q]));  // as stored
          acc[q] += b;
          acc[8 + q] += b * b;
        }
      }
    }
  }
  float* base = a.stats + ((long)r.b * rg.chunks + blockIdx.y) * 2 * N;
  lane_reduce_store<16>(acc, sm, rg, N, base, base + N);
}

dim3 red_dims(const Geo& g, RedGrid rg, int C) {
  (void)C;
  return dim3(g.B, rg.chunks, rg.zb);
}

dim3 red_block(RedGrid rg) { return dim3(rg.vx, rg.py); }

// Element type shared by every tensor source of a launch (the stage dtype),
// or -1 when they disagree (no kernel is instantiated for that).
int common_dt(const VIn& v) {
  if (v.s1.ptr && v.c0 < v.C && v.s1.dtype != v.s0.dtype) return -1;
  return v.s0.dtype;
}

}  // namespace

RedGrid red_grid(const Geo& g, int C) {
  RedGrid rg;
  const int nv = C / 8;
  rg.zb = (nv + 127) / 128;
  rg.vx = (nv + rg.zb - 1) / rg.zb;
  rg.py = 256 / rg.vx;
  const int hw = g.hw();
  int chunks = 2048 / (g.B * rg.zb);
  if (chunks > 128) chunks = 128;
  const int max_chunks = (hw + 4 * rg.py - 1) / (4 * rg.py);
  if (chunks > max_chunks) chunks = max_chunks;
  if (chunks < 1) chunks = 1;
  rg.cp = (hw + chunks - 1) / chunks;
  rg.chunks = (hw + rg.cp - 1) / rg.cp;
  return rg;
}

hipError_t launch_gn_stats_partial(const VIn& x, const Geo& g, RedGrid rg, float* partial,
                                   hipStream_t st, void* copy) {
  const int dt = common_dt(x);
  if (dt < 0) return hipErrorInvalidValue;
  const bool add = x.add != nullptr;
  if (copy && add) return hipErrorInvalidValue;  // the copy is of the tensor as stored
  auto kern = dt == DT_BF16 ? (add ? k_gn_stats_partial<DT_BF16, true>
                                   : k_gn_stats_partial<DT_BF16, false>)
                            : (add ? k_gn_stats_partial<DT_F32, true>
                                   : k_gn_stats_partial<DT_F32, false>);
  hipLaunchKernelGGL(kern, red_dims(g, rg, x.C), red_block(rg), 0, st, x, g, rg, partial, copy);
  return hipGetLastError();
}

hipError_t launch_splitk_finalize_stats(const GemmArgs& a, RedGrid rg, hipStream_t st,
                                        hipEvent_t done) {
  if (a.ksplit < 2 || !a.part || !a.stats || a.gnb || a.out_dtype != DT_BF16 || a.ldo != a.N ||
      a.N % 8 != 0 || (a.resid.s0.ptr && (a.resid.s0.dtype != DT_BF16 || a.resid.add)))
    return hipErrorInvalidValue;
  if (done)
    hipExtLaunchKernelGGL(k_splitk_finalize_stats, red_dims(a.g, rg, a.N), red_block(rg), 0, st,
                          nullptr, done, 0, a, rg);
  else
    hipLaunchKernelGGL(k_splitk_finalize_stats, red_dims(a.g, rg, a.N), red_block(rg), 0, st, a,
                       rg);
  return hipGetLastError();
}

hipError_t launch_gn_stats_finalize(const float* partial, const Geo& g, RedGrid rg, int C,
                                    int G, float eps, const float* gamma, const float* beta,
                                    float* mean, float* rstd, float* scale, float* shift,
                                    hipStream_t st) {
  hipLaunchKernelGGL(k_gn_stats_finalize, dim3(g.B, G), dim3(256), 0, st, partial, g, rg, C, G,
                     eps, gamma, beta, mean, rstd, scale, shift);
  return hipGetLastError();
}

hipError_t launch_gn_apply(const VIn& x, const Geo& g, const float* scale, const float* shift,
                           void* dst0, void* dst1, int dtype, hipStream_t st) {
  const int dt = common_dt(x);
  if (dt < 0 || dt != dtype) return hipErrorInvalidValue;
  const RedGrid rg = red_grid(g, x.C);
  const bool add = x.add != nullptr;
  auto kern = dt == DT_BF16 ? (add ? k_gn_apply<DT_BF16, true> : k_gn_apply<DT_BF16, false>)
                            : (add ? k_gn_apply<DT_F32, true> : k_gn_apply<DT_F32, false>);
  hipLaunchKernelGGL(kern, red_dims(g, rg, x.C), red_block(rg), 0, st, x, g, rg, scale, shift,
                     dst0, dst1);
  return hipGetLastError();
}

hipError_t launch_gn_bwd_partial(const Src& da, const VIn& x, const Geo& g, RedGrid rg,
                                 const float* scale, const float* shift, const float* mean,
                                 const float* rstd, int G, float* partial, hipStream_t st) {
  const int dt = common_dt(x);
  if (dt < 0 || da.dtype != dt) return hipErrorInvalidValue;
  const bool add = x.add != nullptr;
  auto kern = dt == DT_BF16 ? (add ? k_gn_bwd_partial<DT_BF16, true>
                                   : k_gn_bwd_partial<DT_BF16, false>)
                            : (add ? k_gn_bwd_partial<DT_F32, true>
                                   : k_gn_bwd_partial<DT_F32, false>);
  hipLaunchKernelGGL(kern, red_dims(g, rg, x.C), red_block(rg), 0, st, da, x, g, rg, scale,
                     shift, mean, rstd, G, partial);
  return hipGetLastError();
}

hipError_t launch_gn_bwd_finalize(const float* partial, const Geo& g, RedGrid rg, int C,
                                  int G, const float* gamma, float* coef, float* dgamma,
                                  float* dbeta, hipStream_t st) {
  const int nchb = (C + TX - 1) / TX;
  hipLaunchKernelGGL(k_gn_bwd_finalize, dim3(g.B * G + nchb), dim3(256), 0, st, partial, g, rg,
                     C, G, gamma, coef, dgamma, dbeta);
  return hipGetLastError();
}

hipError_t launch_chan_totals(const float* partial, const Geo& g, RedGrid rg, int C, int nslot,
                              float* acc0, float* dup, float* acc1, hipStream_t st) {
  hipLaunchKernelGGL(k_chan_totals, dim3((C + TX - 1) / TX), dim3(256), 0, st, partial,
                     g.B * rg.chunks, C, nslot, acc0, dup, acc1);
  return hipGetLastError();
}

namespace {

template <int DT, bool CHAN, bool ADD0>
auto bwd_apply_kernel(int nf) {
  return nf == 0 ? k_gn_bwd_apply<DT, CHAN, ADD0, 0>
                 : nf == 1 ? k_gn_bwd_apply<DT, CHAN, ADD0, 1> : k_gn_bwd_apply<DT, CHAN, ADD0, 2>;
}

template <int DT>
auto bwd_apply_kernel(bool chan, bool add0, int nf) {
  return chan ? (add0 ? bwd_apply_kernel<DT, true, true>(nf) : bwd_apply_kernel<DT, true, false>(nf))
              : (add0 ? bwd_apply_kernel<DT, false, true>(nf)
                      : bwd_apply_kernel<DT, false, false>(nf));
}

}  // namespace

hipError_t launch_gn_bwd_apply(const Src& da, const VIn& x, const Geo& g, RedGrid rg,
                               const float* scale, const float* shift, const float* mean,
                               const float* rstd, const float* gamma, const float* coef,
                               int G, const GnBwdOut& o, hipStream_t st, hipEvent_t done) {
  const int dt = common_dt(x);
  const bool add0 = o.add0.s0.ptr != nullptr;
  // x is a forward activation (no addend); add0 shares the stage dtype
  if (dt < 0 || da.dtype != dt || x.add || (add0 && common_dt(o.add0) != dt))
    return hipErrorInvalidValue;
  const int nf = (add0 && o.add0.add ? 1 : 0) + (o.add1 ? 1 : 0);
  const bool chan = o.chan_partial != nullptr;
  auto kern = dt == DT_BF16 ? bwd_apply_kernel<DT_BF16>(chan, add0, nf)
                            : bwd_apply_kernel<DT_F32>(chan, add0, nf);
  if (done)  // the event completes with the kernel (no marker packet of its own)
    hipExtLaunchKernelGGL(kern, red_dims(g, rg, x.C), red_block(rg), 0, st, nullptr, done, 0, da, x,
                          g, rg, scale, shift, mean, rstd, gamma, coef, G, o);
  else
    hipLaunchKernelGGL(kern, red_dims(g, rg, x.C), red_block(rg), 0, st, da, x, g, rg, scale,
                       shift, mean, rstd, gamma, coef, G, o);
  return hipGetLastError();
}

hipError_t launch_chan_sum_partial(const VIn& v, const Geo& g, RedGrid rg, float* partial,
                                   hipStream_t st) {
  const int dt = common_dt(v);
  if (dt < 0) return hipErrorInvalidValue;
  const bool add = v.add != nullptr;
  auto kern = dt == DT_BF16 ? (add ? k_chan_sum_partial<DT_BF16, true>
                                   : k_chan_sum_partial<DT_BF16, false>)
                            : (add ? k_chan_sum_partial<DT_F32, true>
                                   : k_chan_sum_partial<DT_F32, false>);
  hipLaunchKernelGGL(kern, red_dims(g, rg, v.C), red_block(rg), 0, st, v, g, rg, partial);
  return hipGetLastError();
}

hipError_t launch_chan_per_image(const float* partial, const Geo& g, RedGrid rg, int C,
                                 int nslot, float* pi, hipStream_t st) {
  hipLaunchKernelGGL(k_chan_per_image, dim3((C + VX - 1) / VX, g.B), dim3(VX, PY), 0, st,
                     partial, rg.chunks, g.B, C, nslot, pi);
  return hipGetLastError();
}

}  // namespace pulse
