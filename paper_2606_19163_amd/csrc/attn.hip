// Multi-head self-attention of the transformer-block stage (gfx950, bf16
// MFMA 16x16x32, fp32 accumulation).  Head dimension 64; L tokens per image
// with L a multiple of 64, at most 4096.  The forward streams keys and
// values through LDS 128 at a time for every L.  The backward holds one
// head's keys and values (or queries and output gradients) in LDS whole up
// to 256 tokens and streams them 64 at a time beyond.  q, k and v are the
// three C-channel thirds of the qkv rows [B*L][3C]; head h owns channels
// [64 h, 64 h + 64) of each third.
//
//   forward : s = q k^T / 8, p = softmax_rows(s), o = p v; the row's
//             log-sum-exp lse = log sum_j exp(s_j) is kept (fp32), not p
//   backward: p is recomputed from q, k and lse; with D = rowsum(do o),
//             dp = do v^T, ds = p (dp - D) / 8, dq = ds k, dk = ds^T q,
//             dv = p^T do.  One kernel per query tile computes dq (and D),
//             one per key tile computes dk and dv from s^T = k q^T, so that
//             neither p nor ds ever goes to memory and no result is
//             accumulated across blocks.
//
// LDS tiles are row-major [rows][64] bf16 with the 16-byte chunks of each
// row permuted (chunk c of row r stored at c ^ swz(r)).  An MFMA operand
// whose k index runs along a tile row is one 16-byte read; one whose k index
// runs down the rows (v in o = p v, k in dq = ds k, q and do in dk and dv)
// comes from two ds_read_b64_tr_b16: within 16 lanes, lane j
// receives element j % 4 of the rows addressed by lanes 4 t + j / 4
// (t = 0..3).  swz keeps both read shapes free of bank conflicts: 16
// consecutive rows of one chunk, and rows {0-3, 8-11} (+16 k) of a 32-byte
// column pair, fall on distinct banks.
#include <hip/hip_runtime.h>

#include "common.hpp"
#include "tkernels.hpp"

namespace pulse {

namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));  // 16 staged bytes

constexpr int HD = 64;        // head dimension
constexpr int QT = 64;        // queries (or keys) per block: 4 waves x 16
constexpr float SCALE = 0.125f;  // 1 / sqrt(64)
constexpr float LOG2E = 1.44269504088896341f;
constexpr float LN2 = 0.693147180559945309f;

__device__ __forceinline__ f32x4 mma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint16_t bf(float f) { return f2bf(f); }

// 2^x as one v_exp_f32: results below 2^-126 flush to zero, which a
// softmax weight relative to its row maximum (at most 1) can lose
__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

// (tile, head, image) of this block.  Blocks are dispatched round-robin
// over the 8 XCDs in linear order; the tiles of one (image, head) read the
// same keys and values, so consecutive dispatch slots of one XCD take
// consecutive tiles (each XCD runs a contiguous range of the linear order)
// and a head's K and V are fetched into one L2, not eight.
__device__ __forceinline__ void tile_of(int& t, int& h, int& b) {
  const int nb = gridDim.x * gridDim.y * gridDim.z;
  const int bid = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
  const int q = nb >> 3, r = nb & 7, x = bid & 7;
  const int lb = x * q + (x < r ? x : r) + (bid >> 3);
  t = lb % gridDim.x;
  const int hb = lb / gridDim.x;
  h = hb % gridDim.y;
  b = hb / gridDim.y;
}

// chunk permutation of tile row r: bit 1 of r -> bit 1, bit 2 -> bit 0,
// bit 3 -> bit 2
__device__ __forceinline__ int swz(int r) {
  return (((r >> 1) & 1) << 1) | ((r >> 2) & 1) | (((r >> 3) & 1) << 2);
}

// element offset of chunk c (8 channels) of row r in a [rows][64] tile
__device__ __forceinline__ int toff(int r, int c) { return r * HD + ((c ^ swz(r)) << 3); }

// rows [0, N) x 64 channels of two token-major tensors (row strides s0,
// s1) into two tiles, 256 threads; every global load is issued before the
// first LDS store, so the block waits for one round trip, not one per chunk
template <int N>
__device__ __forceinline__ void load_tiles(uint16_t* t0, const uint16_t* src0, long s0,
                                           uint16_t* t1, const uint16_t* src1, long s1) {
  constexpr int PER = N * 8 / 256;  // 16-byte chunks per thread and tile
  static_assert(N * 8 % 256 == 0, "whole rounds of 256 chunks");
  uint4 v0[PER], v1[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int e = threadIdx.x + 256 * u;
    const int r = e >> 3, c = e & 7;
    v0[u] = *reinterpret_cast<const uint4*>(src0 + (long)r * s0 + c * 8);
    v1[u] = *reinterpret_cast<const uint4*>(src1 + (long)r * s1 + c * 8);
  }
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int e = threadIdx.x + 256 * u;
    const int r = e >> 3, c = e & 7;
    *reinterpret_cast<uint4*>(t0 + toff(r, c)) = v0[u];
    *reinterpret_cast<uint4*>(t1 + toff(r, c)) = v1[u];
  }
}

// operand of 8 consecutive channels: row r, channels 32 kk + 8 g .. + 7
__device__ __forceinline__ bf16x8 frag_row(const uint16_t* t, int r, int kk, int g) {
  return *reinterpret_cast<const bf16x8*>(t + toff(r, 4 * kk + g));
}

__device__ __forceinline__ v4s rd_tr(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(p));
}

// operand whose k index runs down the tile: k = rows [r0, r0 + 32), the
// other index = channels [d0, d0 + 16); lane (g, j) receives rows
// r0 + 8 g .. + 7 of channel d0 + j
__device__ __forceinline__ bf16x8 frag_tr(const uint16_t* t, int r0, int d0, int lane) {
  const int g = lane >> 4, j = lane & 15;
  const int col = d0 + 4 * (j & 3);
  const int r = r0 + 8 * g + (j >> 2);
  const v4s lo = rd_tr(t + toff(r, col >> 3) + (col & 7));
  const v4s hi = rd_tr(t + toff(r + 4, col >> 3) + (col & 7));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// A wave's strip of 16 rows x W columns (W / 8 chunks per row), chunk c of
// row r at c ^ (r & mask) with mask + 1 the largest power of two <= 16
// dividing the chunk count: 16 rows of one chunk fall on distinct banks.
struct Strip {
  uint16_t* p;
  int chunks, mask;
  __device__ __forceinline__ int off(int r, int c) const {
    return r * chunks * 8 + ((c ^ (r & mask)) << 3);
  }
  // C-layout value of row r, column col
  __device__ __forceinline__ void put(int r, int col, float v) const {
    p[off(r, col >> 3) + (col & 7)] = bf(v);
  }
  // A operand: row m, k = columns 32 ks + 8 g .. + 7
  __device__ __forceinline__ bf16x8 frag(int m, int ks, int g) const {
    return *reinterpret_cast<const bf16x8*>(p + off(m, 4 * ks + g));
  }
};

__device__ __forceinline__ Strip make_strip(uint16_t* p, int width) {
  Strip s;
  s.p = p;
  s.chunks = width / 8;
  const int low = s.chunks & -s.chunks;
  s.mask = (low < 16 ? low : 16) - 1;
  return s;
}

__device__ __forceinline__ float dot8(bf16x8 a, bf16x8 b) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) s += (float)a[i] * (float)b[i];
  return s;
}

// ---------------------------------------------------------------------------
// backward, per query tile: dq = ds k, and D = rowsum(do o) for the key tiles
// ---------------------------------------------------------------------------
template <int L>
__global__ __launch_bounds__(256) void k_attn_bwd_q(const uint16_t* qkv, const uint16_t* o,
                                                    const uint16_t* dout, const float* lse,
                                                    int C, uint16_t* dqkv, float* dsum) {
  __shared__ __attribute__((aligned(16))) uint16_t Ks[L * HD];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[L * HD];  // then the ds strips
  int qt, h, b;
  tile_of(qt, h, b);
  const int H = gridDim.y;
  const long row0 = (long)b * L;
  const long C3 = 3L * C;
  const uint16_t* base = qkv + row0 * C3 + h * HD;
  load_tiles<L>(Ks, base + C, C3, Vs, base + 2 * C, C3);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int m = lane & 15, g = lane >> 4;
  const int q0 = qt * QT + w * 16;
  const long lrow = ((long)b * H + h) * L + q0;  // lse / D index of the wave's first row
  bf16x8 qa[2], da[2];
  float dpart = 0.f;
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    const long r = row0 + q0 + m;
    qa[kk] = *reinterpret_cast<const bf16x8*>(base + (long)(q0 + m) * C3 + 32 * kk + 8 * g);
    da[kk] = *reinterpret_cast<const bf16x8*>(dout + r * C + h * HD + 32 * kk + 8 * g);
    const bf16x8 ov = *reinterpret_cast<const bf16x8*>(o + r * C + h * HD + 32 * kk + 8 * g);
    dpart += dot8(da[kk], ov);
  }
  // D of row m: the lanes m, m + 16, m + 32, m + 48 hold its 64 channels
  dpart += __shfl_xor(dpart, 16, 64);
  dpart += __shfl_xor(dpart, 32, 64);
  if (g == 0) dsum[lrow + m] = dpart;
  float Di[4], li[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    Di[i] = __shfl(dpart, 4 * g + i, 64);
    li[i] = lse[lrow + 4 * g + i];
  }
  __syncthreads();

  constexpr int nb = L / 16;
  f32x4 s[nb], dp[nb];
#pragma unroll
  for (int j = 0; j < nb; ++j) {
    s[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    dp[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      s[j] = mma(qa[kk], frag_row(Ks, 16 * j + m, kk, g), s[j]);
      dp[j] = mma(da[kk], frag_row(Vs, 16 * j + m, kk, g), dp[j]);
    }
  }
  __syncthreads();  // every wave is done with Vs: it now holds the ds strips
  const Strip S = make_strip(Vs + w * 16 * L, L);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < nb; ++j)
    {
      const float p = ex2((s[j][i] * SCALE - li[i]) * LOG2E);
      S.put(4 * g + i, 16 * j + m, p * (dp[j][i] - Di[i]) * SCALE);
    }
  // dq = ds k: A = ds rows (k = key), B = k rows read down the tile
  f32x4 acc[HD / 16];
#pragma unroll
  for (int jd = 0; jd < HD / 16; ++jd) acc[jd] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < L / 32; ++ks) {
    const bf16x8 a = S.frag(m, ks, g);
#pragma unroll
    for (int jd = 0; jd < HD / 16; ++jd)
      acc[jd] = mma(a, frag_tr(Ks, 32 * ks, 16 * jd, lane), acc[jd]);
  }
  const long orow = row0 + q0 + 4 * g;
#pragma unroll
  for (int jd = 0; jd < HD / 16; ++jd)
#pragma unroll
    for (int i = 0; i < 4; ++i) dqkv[(orow + i) * C3 + h * HD + jd * 16 + m] = bf(acc[jd][i]);
}

// ---------------------------------------------------------------------------
// backward, per key tile: wave w owns keys 16 w .. + 15 of the tile and runs
// over the queries 64 at a time: s^T = k q^T, p^T, dp^T = v do^T,
// ds^T = p^T (dp^T - D) / 8, dv += p^T do, dk += ds^T q
// ---------------------------------------------------------------------------
template <int L>
__global__ __launch_bounds__(256) void k_attn_bwd_kv(const uint16_t* qkv, const uint16_t* dout,
                                                     const float* lse, const float* dsum,
                                                     int C, uint16_t* dqkv) {
  __shared__ __attribute__((aligned(16))) uint16_t Qs[L * HD];
  __shared__ __attribute__((aligned(16))) uint16_t dOs[L * HD];
  __shared__ __attribute__((aligned(16))) uint16_t Ws[4][16 * QT];  // p^T, then ds^T, per wave
  int kt, h, b;
  tile_of(kt, h, b);
  const int H = gridDim.y;
  const long row0 = (long)b * L;
  const long C3 = 3L * C;
  const uint16_t* base = qkv + row0 * C3 + h * HD;
  load_tiles<L>(Qs, base, C3, dOs, dout + row0 * C + h * HD, C);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int m = lane & 15, g = lane >> 4;
  const int k0 = kt * QT + w * 16;  // the wave's first key in the image
  const float* lrow = lse + ((long)b * H + h) * L;
  const float* drow = dsum + ((long)b * H + h) * L;
  bf16x8 ka[2], va[2];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    ka[kk] = *reinterpret_cast<const bf16x8*>(base + (long)(k0 + m) * C3 + C + 32 * kk + 8 * g);
    va[kk] =
        *reinterpret_cast<const bf16x8*>(base + (long)(k0 + m) * C3 + 2 * C + 32 * kk + 8 * g);
  }
  // lse and D of the query columns this lane holds: 16 t + m
  float lq[L / 16], dq[L / 16];
#pragma unroll
  for (int t = 0; t < L / 16; ++t) {
    lq[t] = lrow[16 * t + m];
    dq[t] = drow[16 * t + m];
  }
  __syncthreads();

  const Strip W = make_strip(Ws[w], QT);
  f32x4 dv[HD / 16], dk[HD / 16];
#pragma unroll
  for (int jd = 0; jd < HD / 16; ++jd) {
    dv[jd] = f32x4{0.f, 0.f, 0.f, 0.f};
    dk[jd] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
#pragma unroll
  for (int qc = 0; qc < L / QT; ++qc) {
    f32x4 st[4], dpt[4];
#pragma unroll
    for (int jq = 0; jq < 4; ++jq) {
      st[jq] = f32x4{0.f, 0.f, 0.f, 0.f};
      dpt[jq] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int r = qc * QT + 16 * jq + m;
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        st[jq] = mma(ka[kk], frag_row(Qs, r, kk, g), st[jq]);
        dpt[jq] = mma(va[kk], frag_row(dOs, r, kk, g), dpt[jq]);
      }
    }
    // the lane holds keys 4 g + i and query column qc * 64 + 16 jq + m
#pragma unroll
    for (int jq = 0; jq < 4; ++jq)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = ex2((st[jq][i] * SCALE - lq[4 * qc + jq]) * LOG2E);
        st[jq][i] = p;
        dpt[jq][i] = p * (dpt[jq][i] - dq[4 * qc + jq]) * SCALE;
        W.put(4 * g + i, 16 * jq + m, p);
      }
    // dv += p^T do: A = p^T rows (k = query), B = do rows read down the tile
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const bf16x8 a = W.frag(m, ks, g);
#pragma unroll
      for (int jd = 0; jd < HD / 16; ++jd)
        dv[jd] = mma(a, frag_tr(dOs, qc * QT + 32 * ks, 16 * jd, lane), dv[jd]);
    }
    // the strip now takes ds^T (this wave's reads of p^T are issued before)
#pragma unroll
    for (int jq = 0; jq < 4; ++jq)
#pragma unroll
      for (int i = 0; i < 4; ++i) W.put(4 * g + i, 16 * jq + m, dpt[jq][i]);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const bf16x8 a = W.frag(m, ks, g);
#pragma unroll
      for (int jd = 0; jd < HD / 16; ++jd)
        dk[jd] = mma(a, frag_tr(Qs, qc * QT + 32 * ks, 16 * jd, lane), dk[jd]);
    }
  }
  const long krow = row0 + k0 + 4 * g;
#pragma unroll
  for (int jd = 0; jd < HD / 16; ++jd)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const long r = (krow + i) * C3 + h * HD + jd * 16 + m;
      dqkv[r + C] = bf(dk[jd][i]);
      dqkv[r + 2 * C] = bf(dv[jd][i]);
    }
}

// ---------------------------------------------------------------------------
// Backward for longer sequences (L > 256): the same products, streamed
// over 64-token chunks of the other side: key chunks for dq, query chunks
// for dk and dv.  Each chunk is loaded into registers one iteration ahead
// and stored into a single LDS tile per operand at the top of the next
// iteration.
// ---------------------------------------------------------------------------

constexpr int KC = 64;  // tokens per streamed chunk

// the two 16-byte chunks this thread moves of a [64][64] tile
__device__ __forceinline__ void chunk_regs(u32x4 (&v)[2], const uint16_t* src, long stride) {
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int e = threadIdx.x + 256 * u;
    v[u] = *reinterpret_cast<const u32x4*>(src + (long)(e >> 3) * stride + (e & 7) * 8);
  }
}

__device__ __forceinline__ void chunk_store(uint16_t* t, const u32x4 (&v)[2]) {
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int e = threadIdx.x + 256 * u;
    *reinterpret_cast<u32x4*>(t + toff(e >> 3, e & 7)) = v[u];
  }
}

__global__ __launch_bounds__(256) void k_attn_bwd_q_s(const uint16_t* qkv, const uint16_t* o,
                                                      const uint16_t* dout, const float* lse,
                                                      int L, int C, uint16_t* dqkv,
                                                      float* dsum) {
  __shared__ __attribute__((aligned(16))) uint16_t Ks[KC * HD];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[KC * HD];
  __shared__ __attribute__((aligned(16))) uint16_t Ss[4][16 * KC];
  int qt, h, b;
  tile_of(qt, h, b);
  const int H = gridDim.y;
  const long row0 = (long)b * L;
  const long C3 = 3L * C;
  const uint16_t* base = qkv + row0 * C3 + h * HD;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int m = lane & 15, g = lane >> 4;
  const int q0 = qt * QT + w * 16;
  const long lrow = ((long)b * H + h) * L + q0;
  bf16x8 qa[2], da[2];
  float dpart = 0.f;
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    const long r = row0 + q0 + m;
    qa[kk] = *reinterpret_cast<const bf16x8*>(base + (long)(q0 + m) * C3 + 32 * kk + 8 * g);
    da[kk] = *reinterpret_cast<const bf16x8*>(dout + r * C + h * HD + 32 * kk + 8 * g);
    const bf16x8 ov = *reinterpret_cast<const bf16x8*>(o + r * C + h * HD + 32 * kk + 8 * g);
    dpart += dot8(da[kk], ov);
  }
  dpart += __shfl_xor(dpart, 16, 64);
  dpart += __shfl_xor(dpart, 32, 64);
  if (g == 0) dsum[lrow + m] = dpart;
  float Di[4], li[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    Di[i] = __shfl(dpart, 4 * g + i, 64);
    li[i] = lse[lrow + 4 * g + i];
  }
  u32x4 rk[2], rv[2];
  chunk_regs(rk, base + C, C3);
  chunk_regs(rv, base + 2 * C, C3);
  const Strip S = make_strip(Ss[w], KC);
  f32x4 acc[HD / 16];
#pragma unroll
  for (int jd = 0; jd < HD / 16; ++jd) acc[jd] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int nch = L / KC;
  for (int kc = 0; kc < nch; ++kc) {
    __syncthreads();
    chunk_store(Ks, rk);
    chunk_store(Vs, rv);
    __syncthreads();
    {
      const int kn = min(kc + 1, nch - 1);  // unconditional: the wait stays at the store
      chunk_regs(rk, base + (long)kn * KC * C3 + C, C3);
      chunk_regs(rv, base + (long)kn * KC * C3 + 2 * C, C3);
    }
    f32x4 sc[KC / 16], dp[KC / 16];
#pragma unroll
    for (int j = 0; j < KC / 16; ++j) {
      sc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
      dp[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        sc[j] = mma(qa[kk], frag_row(Ks, 16 * j + m, kk, g), sc[j]);
        dp[j] = mma(da[kk], frag_row(Vs, 16 * j + m, kk, g), dp[j]);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < KC / 16; ++j) {
        const float p = ex2((sc[j][i] * SCALE - li[i]) * LOG2E);
        S.put(4 * g + i, 16 * j + m, p * (dp[j][i] - Di[i]) * SCALE);
      }
#pragma unroll
    for (int ks = 0; ks < KC / 32; ++ks) {
      const bf16x8 a = S.frag(m, ks, g);
#pragma unroll
      for (int jd = 0; jd < HD / 16; ++jd)
        acc[jd] = mma(a, frag_tr(Ks, 32 * ks, 16 * jd, lane), acc[jd]);
    }
  }
  const long orow = row0 + q0 + 4 * g;
#pragma unroll
  for (int jd = 0; jd < HD / 16; ++jd)
#pragma unroll
    for (int i = 0; i < 4; ++i) dqkv[(orow + i) * C3 + h * HD + jd * 16 + m] = bf(acc[jd][i]);
}

__global__ __launch_bounds__(256) void k_attn_bwd_kv_s(const uint16_t* qkv, const uint16_t* dout,
                                                       const float* lse, const float* dsum,
                                                       int L, int C, uint16_t* dqkv) {
  __shared__ __attribute__((aligned(16))) uint16_t Qs[KC * HD];
  __shared__ __attribute__((aligned(16))) uint16_t dOs[KC * HD];
  __shared__ __attribute__((aligned(16))) uint16_t Ws[4][16 * KC];
  int kt, h, b;
  tile_of(kt, h, b);
  const int H = gridDim.y;
  const long row0 = (long)b * L;
  const long C3 = 3L * C;
  const uint16_t* base = qkv + row0 * C3 + h * HD;
  const uint16_t* dbase = dout + row0 * C + h * HD;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int m = lane & 15, g = lane >> 4;
  const int k0 = kt * QT + w * 16;
  const float* lrow = lse + ((long)b * H + h) * L;
  const float* drow = dsum + ((long)b * H + h) * L;
  bf16x8 ka[2], va[2];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    ka[kk] = *reinterpret_cast<const bf16x8*>(base + (long)(k0 + m) * C3 + C + 32 * kk + 8 * g);
    va[kk] =
        *reinterpret_cast<const bf16x8*>(base + (long)(k0 + m) * C3 + 2 * C + 32 * kk + 8 * g);
  }
  u32x4 rq[2], rd[2];
  chunk_regs(rq, base, C3);
  chunk_regs(rd, dbase, C);
  const Strip W = make_strip(Ws[w], KC);
  f32x4 dv[HD / 16], dk[HD / 16];
#pragma unroll
  for (int jd = 0; jd < HD / 16; ++jd) {
    dv[jd] = f32x4{0.f, 0.f, 0.f, 0.f};
    dk[jd] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const int nch = L / KC;
  for (int qc = 0; qc < nch; ++qc) {
    // lse and D of the query columns this lane holds in the chunk
    float lq[KC / 16], dq[KC / 16];
#pragma unroll
    for (int jq = 0; jq < KC / 16; ++jq) {
      lq[jq] = lrow[qc * KC + 16 * jq + m];
      dq[jq] = drow[qc * KC + 16 * jq + m];
    }
    __syncthreads();
    chunk_store(Qs, rq);
    chunk_store(dOs, rd);
    __syncthreads();
    {
      const int qn = min(qc + 1, nch - 1);
      chunk_regs(rq, base + (long)qn * KC * C3, C3);
      chunk_regs(rd, dbase + (long)qn * KC * C, C);
    }
    f32x4 st[KC / 16], dpt[KC / 16];
#pragma unroll
    for (int jq = 0; jq < KC / 16; ++jq) {
      st[jq] = f32x4{0.f, 0.f, 0.f, 0.f};
      dpt[jq] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        st[jq] = mma(ka[kk], frag_row(Qs, 16 * jq + m, kk, g), st[jq]);
        dpt[jq] = mma(va[kk], frag_row(dOs, 16 * jq + m, kk, g), dpt[jq]);
      }
    }
#pragma unroll
    for (int jq = 0; jq < KC / 16; ++jq)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = ex2((st[jq][i] * SCALE - lq[jq]) * LOG2E);
        dpt[jq][i] = p * (dpt[jq][i] - dq[jq]) * SCALE;
        W.put(4 * g + i, 16 * jq + m, p);
      }
#pragma unroll
    for (int ks = 0; ks < KC / 32; ++ks) {
      const bf16x8 a = W.frag(m, ks, g);
#pragma unroll
      for (int jd = 0; jd < HD / 16; ++jd)
        dv[jd] = mma(a, frag_tr(dOs, 32 * ks, 16 * jd, lane), dv[jd]);
    }
#pragma unroll
    for (int jq = 0; jq < KC / 16; ++jq)
#pragma unroll
      for (int i = 0; i < 4; ++i) W.put(4 * g + i, 16 * jq + m, dpt[jq][i]);
#pragma unroll
    for (int ks = 0; ks < KC / 32; ++ks) {
      const bf16x8 a = W.frag(m, ks, g);
#pragma unroll
      for (int jd = 0; jd < HD / 16; ++jd)
        dk[jd] = mma(a, frag_tr(Qs, 32 * ks, 16 * jd, lane), dk[jd]);
    }
  }
  const long krow = row0 + k0 + 4 * g;
#pragma unroll
  for (int jd = 0; jd < HD / 16; ++jd)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const long r = (krow + i) * C3 + h * HD + jd * 16 + m;
      dqkv[r + C] = bf(dk[jd][i]);
      dqkv[r + 2 * C] = bf(dv[jd][i]);
    }
}

// ---------------------------------------------------------------------------
// forward, key-split form (any L): block (64-query tile, head, image).  The
// keys stream through LDS 128 at a time and wave w takes keys 32 w .. + 31
// of every chunk for all 64 queries, so each K or V fragment read from LDS
// feeds four MFMAs (one per 16-query block) and p never leaves registers:
//   s^T = k q^T   A = k rows (LDS), B = q (registers); the output lane
//                 (g, m) holds keys 8 g + 4 kb + i of query 16 qb + m
//   o^T += v^T p^T  A = v read down the tile (lane (g, j): keys 8 g + t of
//                 channel 16 db + j), B = p^T (lane (g, m): keys 8 g + t of
//                 query m, t = 4 kb + i: exactly the values the lane holds)
// For the first product to deliver keys 8 g + 4 kb + i on output row 4 g + i
// of block kb, every 32-key group is stored with its rows permuted: key k at
// row (k & 3) | ((k >> 3) & 3) << 2 | ((k >> 2) & 1) << 4, so that rows
// 16 kb .. 16 kb + 15 hold keys 8 (m >> 2) + 4 kb + (m & 3), m = 0..15.
// Every wave keeps a running maximum and sum per query (online softmax); at
// the end the four partial states are merged through LDS.
// ---------------------------------------------------------------------------

constexpr int KS_CHUNK = 128;  // keys per chunk: 4 waves x 32
constexpr int OPAD = 65;       // floats per row of the merge buffers

__device__ __forceinline__ int kperm(int k) {
  return (k & ~31) | (k & 3) | (((k >> 3) & 3) << 2) | (((k >> 2) & 1) << 4);
}

// Chunk staging of the key-split forward.  Thread t moves 16-byte piece
// t % 8 of rows t / 8 + 32 u (u = 0..3) of a 128-row chunk.  Rows 0..63 of
// a chunk always lie in the image (every chunk holds 128 rows but a tail,
// which holds 64); rows 64..127 of a tail are fetched from the image's last
// 64 rows instead (in bounds, never stored).  So every load is
// unconditional, its wait falls at the LDS store of the next iteration, and
// the per-lane offsets are computed once.
__device__ __forceinline__ long piece(long stride) {
  return (long)(threadIdx.x >> 3) * stride + (threadIdx.x & 7) * 8;
}

// chunk [c0, c0 + 128) of two tensors sharing row stride s (pa, pb: row 0
// of each, po: piece(s)); c0 < L
__device__ __forceinline__ void stage2(u32x4 (&a)[4], u32x4 (&b)[4], const uint16_t* pa,
                                       const uint16_t* pb, long s, long po, int c0, int L) {
  const int hi = min(c0 + 64, L - 64);
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const long r = u < 2 ? c0 + 32 * u : hi + 32 * (u - 2);
    a[u] = *reinterpret_cast<const u32x4*>(pa + r * s + po);
    b[u] = *reinterpret_cast<const u32x4*>(pb + r * s + po);
  }
}

// staged rows into two tiles at this thread's offsets oa, ob (row t / 8;
// rows + 32 u sit 32 * 64 elements further: kperm and swz leave the bits
// from 5 up alone); `full`: the chunk holds 128 rows
__device__ __forceinline__ void put2(uint16_t* ta, int oa, uint16_t* tb, int ob,
                                     const u32x4 (&a)[4], const u32x4 (&b)[4], bool full) {
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    if (u >= 2 && !full) break;
    *reinterpret_cast<u32x4*>(ta + oa + 32 * HD * u) = a[u];
    *reinterpret_cast<u32x4*>(tb + ob + 32 * HD * u) = b[u];
  }
}

// Softmax of the key-split forward: each wave keeps, per query, a reference
// r in the log2 domain (scores times SCALE * LOG2E).  Its weights are
// p = 2^(s c - r) <= 2^RGROW: r moves up to the running maximum (and the
// wave's sum and o accumulators are rescaled) only when a score of the
// chunk exceeds it by more than RGROW, decided for the whole wave at once,
// which skips the rescale on most chunks.
constexpr float RGROW = 8.f;

__global__ __launch_bounds__(256, 2) void k_attn_fwd_ks(const uint16_t* qkv, int L, int C,
                                                        uint16_t* o, float* lse) {
  // K and V chunks during the key loop, then the four waves' o^T partials
  __shared__ __attribute__((aligned(16))) float smem[4 * QT * OPAD];
  __shared__ float ml[4][2][QT];
  uint16_t* Ks = reinterpret_cast<uint16_t*>(smem);
  uint16_t* Vs = Ks + KS_CHUNK * HD;
  int qt, h, b;
  tile_of(qt, h, b);
  const int H = gridDim.y;
  const long row0 = (long)b * L;
  const long C3 = 3L * C;
  const uint16_t* base = qkv + row0 * C3 + h * HD;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int m = lane & 15, g = lane >> 4;
  const int q0 = qt * QT;
  const float c = SCALE * LOG2E;

  bf16x8 qa[4][2];
#pragma unroll
  for (int qb = 0; qb < 4; ++qb)
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
      qa[qb][kk] =
          *reinterpret_cast<const bf16x8*>(base + (long)(q0 + 16 * qb + m) * C3 + 32 * kk + 8 * g);

  const long po = piece(C3);
  const int ko = toff(kperm(threadIdx.x >> 3), threadIdx.x & 7);
  const int vo = toff(threadIdx.x >> 3, threadIdx.x & 7);
  u32x4 rk[4], rv[4];
  stage2(rk, rv, base + C, base + 2 * C, C3, po, 0, L);

  float ref[4], lsum[4];  // per lane: the reference and its share of the sum
  f32x4 acc[4][HD / 16];
#pragma unroll
  for (int qb = 0; qb < 4; ++qb) {
    ref[qb] = -INFINITY;
    lsum[qb] = 0.f;
#pragma unroll
    for (int db = 0; db < HD / 16; ++db) acc[qb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const int nch = (L + KS_CHUNK - 1) / KS_CHUNK;
  for (int kc = 0; kc < nch; ++kc) {
    const int rows = min(KS_CHUNK, L - kc * KS_CHUNK);
    __syncthreads();  // every wave is done with the previous chunk
    put2(Ks, ko, Vs, vo, rk, rv, rows == KS_CHUNK);
    __syncthreads();
    stage2(rk, rv, base + C, base + 2 * C, C3, po, min(kc + 1, nch - 1) * KS_CHUNK, L);
    if (32 * w >= rows) continue;  // no keys of this wave in a 64-key tail chunk

    f32x4 sc[4][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const bf16x8 k0 = frag_row(Ks, 32 * w + 16 * kb + m, 0, g);
      const bf16x8 k1 = frag_row(Ks, 32 * w + 16 * kb + m, 1, g);
#pragma unroll
      for (int qb = 0; qb < 4; ++qb)
        sc[qb][kb] = mma(k1, qa[qb][1], mma(k0, qa[qb][0], f32x4{0.f, 0.f, 0.f, 0.f}));
    }
    float mx[4];
    bool grow = false;
#pragma unroll
    for (int qb = 0; qb < 4; ++qb) {
      float v = fmaxf(fmaxf(fmaxf(sc[qb][0][0], sc[qb][0][1]), fmaxf(sc[qb][0][2], sc[qb][0][3])),
                      fmaxf(fmaxf(sc[qb][1][0], sc[qb][1][1]), fmaxf(sc[qb][1][2], sc[qb][1][3])));
      v = fmaxf(v, __shfl_xor(v, 16, 64));
      v = fmaxf(v, __shfl_xor(v, 32, 64));
      mx[qb] = v * c;
      grow |= mx[qb] > ref[qb] + RGROW;
    }
    if (__any(grow)) {
#pragma unroll
      for (int qb = 0; qb < 4; ++qb) {
        const float nr = fmaxf(ref[qb], mx[qb]);
        const float alpha = ex2(ref[qb] - nr);  // 0 on the wave's first chunk
        ref[qb] = nr;
        lsum[qb] *= alpha;
#pragma unroll
        for (int db = 0; db < HD / 16; ++db)
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[qb][db][i] *= alpha;
      }
    }
    bf16x8 pb[4];
#pragma unroll
    for (int qb = 0; qb < 4; ++qb)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float e = ex2(fmaf(sc[qb][kb][i], c, -ref[qb]));
          lsum[qb] += e;
          pb[qb][4 * kb + i] = (__bf16)e;
        }
#pragma unroll
    for (int db = 0; db < HD / 16; ++db) {
      const bf16x8 va = frag_tr(Vs, 32 * w, 16 * db, lane);
#pragma unroll
      for (int qb = 0; qb < 4; ++qb) acc[qb][db] = mma(va, pb[qb], acc[qb][db]);
    }
  }

  // merge: R = max_w r_w, l = sum_w l_w 2^(r_w - R), o = sum_w f_w o_w with
  // f_w = 2^(r_w - R) / l; lse = (R + log2 l) ln 2
#pragma unroll
  for (int qb = 0; qb < 4; ++qb) {
    lsum[qb] += __shfl_xor(lsum[qb], 16, 64);
    lsum[qb] += __shfl_xor(lsum[qb], 32, 64);
  }
  if (g == 0) {
#pragma unroll
    for (int qb = 0; qb < 4; ++qb) {
      ml[w][0][16 * qb + m] = ref[qb];
      ml[w][1][16 * qb + m] = lsum[qb];
    }
  }
  __syncthreads();  // also: every wave is done with the K and V chunks
  float* part = smem + w * QT * OPAD;
#pragma unroll
  for (int qb = 0; qb < 4; ++qb) {
    const int q = 16 * qb + m;
    float R = ml[0][0][q];
#pragma unroll
    for (int v = 1; v < 4; ++v) R = fmaxf(R, ml[v][0][q]);
    float l = 0.f;
#pragma unroll
    for (int v = 0; v < 4; ++v) l += ml[v][1][q] * ex2(ml[v][0][q] - R);
    const float f = ex2(ref[qb] - R) / l;
#pragma unroll
    for (int db = 0; db < HD / 16; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) part[q * OPAD + 16 * db + 4 * g + i] = acc[qb][db][i] * f;
    if (w == 0 && g == 0)
      lse[((long)b * H + h) * L + q0 + q] = (R + log2f(l)) * LN2;
  }
  __syncthreads();
  // 64 queries x 64 channels: thread t writes 16 channels of query t / 4
  {
    const int q = threadIdx.x >> 2, d0 = (threadIdx.x & 3) * 16;
    uint32_t pk[8];
#pragma unroll
    for (int j = 0; j < 16; j += 2) {
      const int ix = q * OPAD + d0 + j;
      const float v0 = smem[ix] + smem[QT * OPAD + ix] + smem[2 * QT * OPAD + ix] +
                       smem[3 * QT * OPAD + ix];
      const float v1 = smem[ix + 1] + smem[QT * OPAD + ix + 1] + smem[2 * QT * OPAD + ix + 1] +
                       smem[3 * QT * OPAD + ix + 1];
      pk[j / 2] = (uint32_t)bf(v0) | ((uint32_t)bf(v1) << 16);
    }
    uint4* dst = reinterpret_cast<uint4*>(o + (row0 + q0 + q) * C + h * HD + d0);
    dst[0] = uint4{pk[0], pk[1], pk[2], pk[3]};
    dst[1] = uint4{pk[4], pk[5], pk[6], pk[7]};
  }
}

}  // namespace

bool attn_fits(int L, int C, int heads) {
  return L >= QT && L % QT == 0 && L <= ATTN_LMAX && C == heads * HD;
}

template <int L>
static hipError_t attn_bwd_t(const void* qkv, const void* o, const void* dout, const float* lse,
                             int B, int C, int heads, void* dqkv, float* dsum, hipStream_t st) {
  hipLaunchKernelGGL(k_attn_bwd_q<L>, dim3(L / QT, heads, B), dim3(256), 0, st,
                     static_cast<const uint16_t*>(qkv), static_cast<const uint16_t*>(o),
                     static_cast<const uint16_t*>(dout), lse, C, static_cast<uint16_t*>(dqkv),
                     dsum);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_attn_bwd_kv<L>, dim3(L / QT, heads, B), dim3(256), 0, st,
                     static_cast<const uint16_t*>(qkv), static_cast<const uint16_t*>(dout), lse,
                     dsum, C, static_cast<uint16_t*>(dqkv));
  return hipGetLastError();
}

hipError_t launch_attn_fwd(const void* qkv, int B, int L, int C, int heads, void* o, float* lse,
                           hipStream_t st) {
  if (!attn_fits(L, C, heads)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_attn_fwd_ks, dim3(L / QT, heads, B), dim3(256), 0, st,
                     static_cast<const uint16_t*>(qkv), L, C, static_cast<uint16_t*>(o), lse);
  return hipGetLastError();
}

hipError_t launch_attn_bwd(const void* qkv, const void* o, const void* dout, const float* lse,
                           int B, int L, int C, int heads, void* dqkv, float* dsum,
                           hipStream_t st) {
  if (!attn_fits(L, C, heads)) return hipErrorInvalidValue;
  switch (L) {
    case 64: return attn_bwd_t<64>(qkv, o, dout, lse, B, C, heads, dqkv, dsum, st);
    case 128: return attn_bwd_t<128>(qkv, o, dout, lse, B, C, heads, dqkv, dsum, st);
    case 192: return attn_bwd_t<192>(qkv, o, dout, lse, B, C, heads, dqkv, dsum, st);
    case 256: return attn_bwd_t<256>(qkv, o, dout, lse, B, C, heads, dqkv, dsum, st);
    default: {
      hipLaunchKernelGGL(k_attn_bwd_q_s, dim3(L / QT, heads, B), dim3(256), 0, st,
                         static_cast<const uint16_t*>(qkv), static_cast<const uint16_t*>(o),
                         static_cast<const uint16_t*>(dout), lse, L, C,
                         static_cast<uint16_t*>(dqkv), dsum);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL(k_attn_bwd_kv_s, dim3(L / QT, heads, B), dim3(256), 0, st,
                         static_cast<const uint16_t*>(qkv), static_cast<const uint16_t*>(dout),
                         lse, dsum, L, C, static_cast<uint16_t*>(dqkv));
      return hipGetLastError();
    }
  }
}

}  // namespace pulse
