// GroupNorm + SiLU forward/backward and per-channel reductions over NHWC
// activations (gfx950).  All of it is HBM-bound streaming: a block owns one
// image, one chunk of pixels and 64 channel vectors of 8 channels; its 256
// threads are 64 channel vectors x 4 pixel lanes, so each pixel row of a
// block is one contiguous, coalesced read.  Reductions are deterministic:
// fixed per-thread order, a fixed LDS tree, per-(image, chunk) partials and
// a finalize that sums them in a fixed order (group sums in fp64).
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

// Sum the pixel lanes of NV values per thread through LDS (fixed order) and
// let lane 0 write 8 of them to out0 (and the next 8 to out1).
template <int NV>
__device__ __forceinline__ void lane_reduce_store(float (&v)[NV], float* sm, RedGrid rg,
                                                  bool active, float* out0, float* out1) {
  const int tx = threadIdx.x, ty = threadIdx.y;
#pragma unroll
  for (int i = 0; i < NV; ++i) sm[(ty * rg.vx + tx) * NV + i] = v[i];
  __syncthreads();
  if (ty == 0 && active) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      float s = sm[tx * NV + i];
      for (int y = 1; y < rg.py; ++y) s += sm[(y * rg.vx + tx) * NV + i];
      v[i] = s;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) out0[i] = v[i];
    if (out1) {
#pragma unroll
      for (int i = 0; i < 8 && 8 + i < NV; ++i) out1[i] = v[8 + i];
    }
  }
}

__global__ __launch_bounds__(256) void k_gn_stats_partial(VIn x, Geo g, RedGrid rg,
                                                          float* partial) {
  __shared__ float sm[256 * 16];
  const Range r = block_range(g, rg, x.C);
  float acc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.f;
  if (r.active) {
    // four pixels per iteration keep four loads in flight per thread
    for (int p = r.p0 + threadIdx.y; p < r.p1; p += 4 * rg.py) {
      float f[4][8];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int pu = p + u * rg.py;
        if (pu < r.p1) {
          ld8v(x, (long)r.b * g.hw() + pu, r.c, f[u]);
        } else {
#pragma unroll
          for (int i = 0; i < 8; ++i) f[u][i] = 0.f;
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          acc[i] += f[u][i];
          acc[8 + i] += f[u][i] * f[u][i];
        }
    }
  }
  float* base = partial + ((long)r.b * rg.chunks + blockIdx.y) * 2 * x.C;
  lane_reduce_store<16>(acc, sm, rg, r.active, base + r.c, base + x.C + r.c);
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
  for (int i = threadIdx.x; i < rg.chunks * cg; i += 256) {
    const int ch = i / cg;
    const int c = gi * cg + (i - ch * cg);
    const float* base = partial + ((long)b * rg.chunks + ch) * 2 * C;
    S += base[c];
    Q += base[C + c];
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

__global__ __launch_bounds__(256) void k_gn_apply(VIn x, Geo g, const float* scale,
                                                  const float* shift, void* dst0, void* dst1,
                                                  int dtype) {
  const int NV = x.C / 8;
  const long total = g.pixels() * NV;
  const int HW = g.hw();
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (long)gridDim.x * blockDim.x) {
    const long pix = i / NV;
    const int c = (int)(i - pix * NV) * 8;
    const int b = (int)(pix / HW);
    float f[8];
    ld8v(x, pix, c, f);
    const float4* sc = reinterpret_cast<const float4*>(scale + (long)b * x.C + c);
    const float4* sh = reinterpret_cast<const float4*>(shift + (long)b * x.C + c);
    const float4 s0 = sc[0], s1 = sc[1], h0 = sh[0], h1 = sh[1];
    const float ss[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
    const float hh[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
#pragma unroll
    for (int j = 0; j < 8; ++j) f[j] = silu_f(f[j] * ss[j] + hh[j]);
    if (c < x.c0)
      st8(dst0, dtype, x.c0, pix, c, f);
    else
      st8(dst1, dtype, x.C - x.c0, pix, c - x.c0, f);
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

__global__ __launch_bounds__(256) void k_gn_bwd_partial(Src da, VIn x, Geo g,
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
    for (int p = r.p0 + threadIdx.y; p < r.p1; p += rg.py) {
      float f[1][8], d[1][8];
#pragma unroll
      for (int u = 0; u < 1; ++u) {
        const int pu = p + u * rg.py;
        if (pu < r.p1) {
          const long pix = (long)r.b * g.hw() + pu;
          ld8v(x, pix, r.c, f[u]);
          ld8(da, pix, r.c, d[u]);
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j) f[u][j] = d[u][j] = 0.f;
        }
      }
#pragma unroll
      for (int u = 0; u < 1; ++u)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float z = f[u][j] * k.sc[j] + k.sh[j];
          const float dz = d[u][j] * dsilu_f(z);
          const float xh = (f[u][j] - k.mu[j]) * k.rs[j];
          acc[j] += dz;
          acc[8 + j] += dz * xh;
        }
    }
  }
  float* base = partial + ((long)r.b * rg.chunks + blockIdx.y) * 2 * x.C;
  lane_reduce_store<16>(acc, sm, rg, r.active, base + r.c, base + x.C + r.c);
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
// acc0 (and dup), slot 1 to acc1.  A 1024-thread block holds 16 channels x
// 64 row lanes; lane y sums the (image, chunk) rows y, y+64, ... and the
// lanes meet in a fixed LDS tree.
constexpr int TX = 16, TY = 64;

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
    int i = ty;
    for (; i + TY < rows; i += 2 * TY) {
      const float a0 = base[i * stride], a1 = base[(i + TY) * stride];
      const float e0 = nslot > 1 ? base[i * stride + C] : 0.f;
      const float e1 = nslot > 1 ? base[(i + TY) * stride + C] : 0.f;
      s0 += a0;
      s0 += a1;
      s1 += e0;
      s1 += e1;
    }
    for (; i < rows; i += TY) {
      s0 += base[i * stride];
      if (nslot > 1) s1 += base[i * stride + C];
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

__global__ __launch_bounds__(1024) void k_chan_totals(const float* partial, int rows, int C,
                                                      int nslot, float* acc0, float* dup,
                                                      float* acc1) {
  __shared__ float sm[2][TY][TX];
  chan_totals_block(partial, rows, C, nslot, blockIdx.x, acc0, dup, acc1, sm);
}

// Fixed-order sum of two fp64 values over a 1024-thread block.
__device__ __forceinline__ void block_sum2_1k(double& a, double& b, double* sm) {
  const int t = threadIdx.x;
  sm[t] = a;
  sm[1024 + t] = b;
  __syncthreads();
  for (int off = 512; off > 0; off >>= 1) {
    if (t < off) {
      sm[t] += sm[t + off];
      sm[1024 + t] += sm[1024 + t + off];
    }
    __syncthreads();
  }
  a = sm[0];
  b = sm[1024];
}

// GroupNorm backward finalize in one launch of 1024-thread blocks: blocks
// [0, ceil(C/16)) add dbeta (sum dz) and dgamma (sum dz * xhat) over every
// image and chunk; the remaining B*G blocks each reduce one (image, group)
// to coef = (sum gamma*dz, sum gamma*dz*xhat) / count.
__global__ __launch_bounds__(1024) void k_gn_bwd_finalize(const float* partial, Geo g,
                                                          RedGrid rg, int C, int G,
                                                          const float* gamma, float* coef,
                                                          float* dgamma, float* dbeta) {
  __shared__ float smc[2][TY][TX];
  __shared__ double sm[2048];
  const int nchb = (C + TX - 1) / TX;
  if ((int)blockIdx.x < nchb) {
    chan_totals_block(partial, g.B * rg.chunks, C, 2, blockIdx.x, dbeta, nullptr, dgamma, smc);
    return;
  }
  const int q = blockIdx.x - nchb;
  const int b = q / G, gi = q - b * G;
  const int cg = C / G;
  double S1 = 0.0, S2 = 0.0;
  for (int i = threadIdx.x; i < rg.chunks * cg; i += 1024) {
    const int ch = i / cg;
    const int c = gi * cg + (i - ch * cg);
    const float* base = partial + ((long)b * rg.chunks + ch) * 2 * C;
    S1 += (double)gamma[c] * base[c];
    S2 += (double)gamma[c] * base[C + c];
  }
  block_sum2_1k(S1, S2, sm);
  if (threadIdx.x == 0) {
    const double cnt = (double)g.hw() * cg;
    coef[(b * G + gi) * 2 + 0] = (float)(S1 / cnt);
    coef[(b * G + gi) * 2 + 1] = (float)(S2 / cnt);
  }
}

// CHAN: the output's per-chunk channel sums are written (the timestep-
// embedding gradient); ADD: the addends add0/add1 exist.  Each instance keeps
// only the registers it needs.
template <bool CHAN, bool ADD>
__global__ __launch_bounds__(256) void k_gn_bwd_apply(Src da, VIn x, Geo g,
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
    for (int p = r.p0 + threadIdx.y; p < r.p1; p += rg.py) {
      const long pix = (long)r.b * g.hw() + p;
      float f[8], d[8], out[8];
      ld8v(x, pix, r.c, f);
      ld8(da, pix, r.c, d);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float dz = d[j] * dsilu_f(f[j] * sc[j] + sh[j]);
        out[j] = A[j] * dz + (Bq[j] * f[j] + Cq[j]);
      }
      if (ADD && o.add0.s0.ptr) {
        float e[8];
        ld8v(o.add0, pix, r.c, e);
#pragma unroll
        for (int j = 0; j < 8; ++j) out[j] += e[j];
      }
      if (ADD && o.add1) {
        const float4* ap = reinterpret_cast<const float4*>(o.add1 + pix * C + r.c);
        const float4 a0 = ap[0], a1 = ap[1];
        out[0] += a0.x; out[1] += a0.y; out[2] += a0.z; out[3] += a0.w;
        out[4] += a1.x; out[5] += a1.y; out[6] += a1.z; out[7] += a1.w;
      }
      if (r.c < o.c_split)
        st8(o.dst0, o.dtype0, o.c_split, pix, r.c, out);
      else
        st8(o.dst1, o.dtype1, C - o.c_split, pix, r.c - o.c_split, out);
      if (CHAN) {
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] += out[j];
      }
    }
  }
  if (CHAN) {
    float* base = o.chan_partial + ((long)r.b * rg.chunks + blockIdx.y) * 2 * C;
    lane_reduce_store<8>(acc, sm, rg, r.active, base + r.c, nullptr);
  }
}

__global__ __launch_bounds__(256) void k_chan_sum_partial(VIn v, Geo g, RedGrid rg,
                                                          float* partial) {
  __shared__ float sm[256 * 8];
  const Range r = block_range(g, rg, v.C);
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
  if (r.active) {
    for (int p = r.p0 + threadIdx.y; p < r.p1; p += rg.py) {
      float f[8];
      ld8v(v, (long)r.b * g.hw() + p, r.c, f);
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] += f[j];
    }
  }
  float* base = partial + ((long)r.b * rg.chunks + blockIdx.y) * 2 * v.C;
  lane_reduce_store<8>(acc, sm, rg, r.active, base + r.c, nullptr);
}

dim3 red_dims(const Geo& g, RedGrid rg, int C) {
  (void)C;
  return dim3(g.B, rg.chunks, rg.zb);
}

dim3 red_block(RedGrid rg) { return dim3(rg.vx, rg.py); }

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
                                   hipStream_t st) {
  hipLaunchKernelGGL(k_gn_stats_partial, red_dims(g, rg, x.C), red_block(rg), 0, st, x, g, rg,
                     partial);
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
  const long total = g.pixels() * (x.C / 8);
  long blocks = (total + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(k_gn_apply, dim3((unsigned)blocks), dim3(256), 0, st, x, g, scale, shift,
                     dst0, dst1, dtype);
  return hipGetLastError();
}

hipError_t launch_gn_bwd_partial(const Src& da, const VIn& x, const Geo& g, RedGrid rg,
                                 const float* scale, const float* shift, const float* mean,
                                 const float* rstd, int G, float* partial, hipStream_t st) {
  hipLaunchKernelGGL(k_gn_bwd_partial, red_dims(g, rg, x.C), red_block(rg), 0, st, da, x, g, rg,
                     scale, shift, mean, rstd, G, partial);
  return hipGetLastError();
}

hipError_t launch_gn_bwd_finalize(const float* partial, const Geo& g, RedGrid rg, int C,
                                  int G, const float* gamma, float* coef, float* dgamma,
                                  float* dbeta, hipStream_t st) {
  const int nchb = (C + TX - 1) / TX;
  hipLaunchKernelGGL(k_gn_bwd_finalize, dim3(nchb + g.B * G), dim3(1024), 0, st, partial, g, rg,
                     C, G, gamma, coef, dgamma, dbeta);
  return hipGetLastError();
}

hipError_t launch_chan_totals(const float* partial, const Geo& g, RedGrid rg, int C, int nslot,
                              float* acc0, float* dup, float* acc1, hipStream_t st) {
  hipLaunchKernelGGL(k_chan_totals, dim3((C + TX - 1) / TX), dim3(1024), 0, st, partial,
                     g.B * rg.chunks, C, nslot, acc0, dup, acc1);
  return hipGetLastError();
}

hipError_t launch_gn_bwd_apply(const Src& da, const VIn& x, const Geo& g, RedGrid rg,
                               const float* scale, const float* shift, const float* mean,
                               const float* rstd, const float* gamma, const float* coef,
                               int G, const GnBwdOut& o, hipStream_t st) {
  const bool chan = o.chan_partial != nullptr, add = o.add0.s0.ptr || o.add1;
  auto kern = chan ? (add ? k_gn_bwd_apply<true, true> : k_gn_bwd_apply<true, false>)
                   : (add ? k_gn_bwd_apply<false, true> : k_gn_bwd_apply<false, false>);
  hipLaunchKernelGGL(kern, red_dims(g, rg, x.C), red_block(rg), 0, st, da, x, g, rg,
                     scale, shift, mean, rstd, gamma, coef, G, o);
  return hipGetLastError();
}

hipError_t launch_chan_sum_partial(const VIn& v, const Geo& g, RedGrid rg, float* partial,
                                   hipStream_t st) {
  hipLaunchKernelGGL(k_chan_sum_partial, red_dims(g, rg, v.C), red_block(rg), 0, st, v, g, rg,
                     partial);
  return hipGetLastError();
}

hipError_t launch_chan_per_image(const float* partial, const Geo& g, RedGrid rg, int C,
                                 int nslot, float* pi, hipStream_t st) {
  hipLaunchKernelGGL(k_chan_per_image, dim3((C + VX - 1) / VX, g.B), dim3(VX, PY), 0, st,
                     partial, rg.chunks, g.B, C, nslot, pi);
  return hipGetLastError();
}

}  // namespace pulse
