// Multi-head self-attention of the transformer-block stage (gfx950, bf16
// MFMA 16x16x32, fp32 accumulation).  Head dimension 64; L tokens per image
// with L a multiple of 64 and at most 256, so a head's keys and values fit
// in LDS whole.  q, k and v are the three C-channel thirds of the qkv rows
// [B*L][3C]; head h owns channels [64 h, 64 h + 64) of each third.
//
//   forward  : s = q k^T / 8, p = softmax_rows(s), o = p v; p is kept (bf16)
//              for the backward pass
//   backward : dp = do v^T, ds = p (dp - rowsum(p dp)) / 8,
//              dq = ds k, dk = ds^T q, dv = p^T do
//
// Every product runs on MFMA with operands read from LDS as 16-byte rows of
// 8 consecutive k values.  Operands whose k index is not the contiguous one
// in memory (v and k in the forward/backward products over keys, p^T, ds^T,
// q^T and do^T) are transposed on their way into LDS.
#include <hip/hip_runtime.h>

#include "common.hpp"
#include "tkernels.hpp"

namespace pulse {

namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

constexpr int HD = 64;        // head dimension
constexpr int QT = 64;        // queries (or keys) per block: 4 waves x 16
constexpr int LMAX = 256;     // tokens per image, at most
constexpr float SCALE = 0.125f;  // 1 / sqrt(64)

__device__ __forceinline__ f32x4 mma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// 8 consecutive bf16 at p (16-byte aligned) as an MFMA operand
__device__ __forceinline__ bf16x8 ld8lds(const uint16_t* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}

// Reduce over the 16 lanes that share lane / 16 (one row of a 16x16 block).
__device__ __forceinline__ float row_max16(float v) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float row_sum16(float v) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Copy rows [r0, r0 + n) of 64 bf16 (a head's channels) from a token-major
// tensor into LDS rows of 64 (row stride 64 elements).
__device__ __forceinline__ void load_rows(uint16_t* dst, const uint16_t* src, long stride, int n) {
  for (int e = threadIdx.x; e < n * 8; e += blockDim.x) {
    const int r = e >> 3, c = (e & 7) * 8;
    *reinterpret_cast<uint4*>(dst + r * HD + c) =
        *reinterpret_cast<const uint4*>(src + (long)r * stride + c);
  }
}

// Transposed copy: the same rows land as columns of dst [64][ld] (dst[c][r]).
__device__ __forceinline__ void load_rows_t(uint16_t* dst, int ld, const uint16_t* src,
                                            long stride, int n) {
  for (int e = threadIdx.x; e < n * 8; e += blockDim.x) {
    const int r = e >> 3, c = (e & 7) * 8;
    const uint4 q = *reinterpret_cast<const uint4*>(src + (long)r * stride + c);
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      dst[(c + 2 * i) * ld + r] = (uint16_t)(w[i] & 0xffffu);
      dst[(c + 2 * i + 1) * ld + r] = (uint16_t)(w[i] >> 16);
    }
  }
}

// Transposed copy of an L x L bf16 matrix block: rows [0, L) and columns
// [c0, c0 + 64) of src (row stride L) into dst[64][L] (dst[c][r]).
__device__ __forceinline__ void load_cols_t(uint16_t* dst, const uint16_t* src, int L, int c0) {
  for (int e = threadIdx.x; e < L * 8; e += blockDim.x) {
    const int r = e >> 3, c = (e & 7) * 8;
    const uint4 q = *reinterpret_cast<const uint4*>(src + (long)r * L + c0 + c);
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      dst[(c + 2 * i) * L + r] = (uint16_t)(w[i] & 0xffffu);
      dst[(c + 2 * i + 1) * L + r] = (uint16_t)(w[i] >> 16);
    }
  }
}

__device__ __forceinline__ uint16_t bf(float f) { return f2bf(f); }

// ---------------------------------------------------------------------------
// forward: block (query tile, head, image); wave w owns queries 16 w .. +15
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_attn_fwd(const uint16_t* qkv, int L, int C,
                                                  uint16_t* o, uint16_t* pbuf) {
  __shared__ __attribute__((aligned(16))) uint16_t Qs[QT * HD];
  __shared__ __attribute__((aligned(16))) uint16_t Ks[LMAX * HD];
  __shared__ __attribute__((aligned(16))) uint16_t VT[HD * LMAX];   // [d][key]
  __shared__ __attribute__((aligned(16))) uint16_t Ps[4][16 * LMAX];  // per wave [q][key]
  const int qt = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int H = gridDim.y;
  const long row0 = (long)b * L;
  const long C3 = 3L * C;
  const uint16_t* base = qkv + row0 * C3 + h * HD;
  load_rows(Qs, base + (long)qt * QT * C3, C3, QT);
  load_rows(Ks, base + C, C3, L);
  load_rows_t(VT, L, base + 2 * C, C3, L);
  __syncthreads();

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int m = lane & 15, g = lane >> 4;
  const int nb = L / 16;
  f32x4 s[LMAX / 16];
#pragma unroll
  for (int j = 0; j < LMAX / 16; ++j) s[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < HD / 32; ++ks) {
    const bf16x8 a = ld8lds(Qs + (w * 16 + m) * HD + ks * 32 + g * 8);
#pragma unroll
    for (int j = 0; j < LMAX / 16; ++j)
      if (j < nb) s[j] = mma(a, ld8lds(Ks + (j * 16 + m) * HD + ks * 32 + g * 8), s[j]);
  }
  // softmax of rows 4 g + i (the lane holds column m of every 16-key block)
  uint16_t* P = Ps[w];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < LMAX / 16; ++j)
      if (j < nb) mx = fmaxf(mx, s[j][i] * SCALE);
    mx = row_max16(mx);
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < LMAX / 16; ++j)
      if (j < nb) {
        const float e = __expf(s[j][i] * SCALE - mx);
        s[j][i] = e;
        sum += e;
      }
    sum = row_sum16(sum);
    const float inv = 1.0f / sum;
#pragma unroll
    for (int j = 0; j < LMAX / 16; ++j)
      if (j < nb) P[(4 * g + i) * L + j * 16 + m] = bf(s[j][i] * inv);
  }
  __syncthreads();
  // o = p v: A = p rows (k = key), B = v^T rows (k = key)
  f32x4 acc[HD / 16];
#pragma unroll
  for (int jd = 0; jd < HD / 16; ++jd) acc[jd] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int ks = 0; ks < L / 32; ++ks) {
    const bf16x8 a = ld8lds(P + m * L + ks * 32 + g * 8);
#pragma unroll
    for (int jd = 0; jd < HD / 16; ++jd)
      acc[jd] = mma(a, ld8lds(VT + (jd * 16 + m) * L + ks * 32 + g * 8), acc[jd]);
  }
  const long q0 = row0 + (long)qt * QT + w * 16;
#pragma unroll
  for (int jd = 0; jd < HD / 16; ++jd)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      o[(q0 + 4 * g + i) * C + h * HD + jd * 16 + m] = bf(acc[jd][i]);
  // keep p for the backward pass: [b][h][q][key]
  uint16_t* pg = pbuf + (((long)b * H + h) * L + (long)qt * QT + w * 16) * L;
  for (int e = lane; e < 16 * L / 8; e += 64)
    *reinterpret_cast<uint4*>(pg + e * 8) = *reinterpret_cast<const uint4*>(P + e * 8);
}

// ---------------------------------------------------------------------------
// backward, per query tile: dp = do v^T, ds = p (dp - rowsum(p dp)) / 8,
// dq = ds k; ds kept (bf16) for the key-side kernel
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_attn_bwd_q(const uint16_t* qkv, const uint16_t* dout,
                                                    const uint16_t* pbuf, int L, int C,
                                                    uint16_t* dqkv, uint16_t* dsbuf) {
  __shared__ __attribute__((aligned(16))) uint16_t dOs[QT * HD];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[LMAX * HD];    // [key][d]
  __shared__ __attribute__((aligned(16))) uint16_t KT[HD * LMAX];    // [d][key]
  __shared__ __attribute__((aligned(16))) uint16_t Ss[4][16 * LMAX];  // per wave ds [q][key]
  const int qt = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int H = gridDim.y;
  const long row0 = (long)b * L;
  const long C3 = 3L * C;
  const uint16_t* base = qkv + row0 * C3 + h * HD;
  load_rows(dOs, dout + (row0 + (long)qt * QT) * C + h * HD, C, QT);
  load_rows(Vs, base + 2 * C, C3, L);
  load_rows_t(KT, L, base + C, C3, L);
  __syncthreads();

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int m = lane & 15, g = lane >> 4;
  const int nb = L / 16;
  f32x4 dp[LMAX / 16];
#pragma unroll
  for (int j = 0; j < LMAX / 16; ++j) dp[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < HD / 32; ++ks) {
    const bf16x8 a = ld8lds(dOs + (w * 16 + m) * HD + ks * 32 + g * 8);
#pragma unroll
    for (int j = 0; j < LMAX / 16; ++j)
      if (j < nb) dp[j] = mma(a, ld8lds(Vs + (j * 16 + m) * HD + ks * 32 + g * 8), dp[j]);
  }
  const long q0 = (long)qt * QT + w * 16;  // within the image
  const uint16_t* pr = pbuf + (((long)b * H + h) * L + q0) * L;
  uint16_t* S = Ss[w];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 4 * g + i;
    float pv[LMAX / 16];
    float t = 0.f;
#pragma unroll
    for (int j = 0; j < LMAX / 16; ++j)
      if (j < nb) {
        pv[j] = bf2f(pr[(long)r * L + j * 16 + m]);
        t += pv[j] * dp[j][i];
      }
    t = row_sum16(t);
#pragma unroll
    for (int j = 0; j < LMAX / 16; ++j)
      if (j < nb) S[r * L + j * 16 + m] = bf(pv[j] * (dp[j][i] - t) * SCALE);
  }
  __syncthreads();
  // dq = ds k: A = ds rows (k = key), B = k^T rows (k = key)
  f32x4 acc[HD / 16];
#pragma unroll
  for (int jd = 0; jd < HD / 16; ++jd) acc[jd] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int ks = 0; ks < L / 32; ++ks) {
    const bf16x8 a = ld8lds(S + m * L + ks * 32 + g * 8);
#pragma unroll
    for (int jd = 0; jd < HD / 16; ++jd)
      acc[jd] = mma(a, ld8lds(KT + (jd * 16 + m) * L + ks * 32 + g * 8), acc[jd]);
  }
#pragma unroll
  for (int jd = 0; jd < HD / 16; ++jd)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      dqkv[(row0 + q0 + 4 * g + i) * C3 + h * HD + jd * 16 + m] = bf(acc[jd][i]);
  uint16_t* dg = dsbuf + (((long)b * H + h) * L + q0) * L;
  for (int e = lane; e < 16 * L / 8; e += 64)
    *reinterpret_cast<uint4*>(dg + e * 8) = *reinterpret_cast<const uint4*>(S + e * 8);
}

// ---------------------------------------------------------------------------
// backward, per key tile: dv = p^T do, dk = ds^T q; wave w owns keys
// 16 w .. +15 of the tile
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_attn_bwd_kv(const uint16_t* qkv, const uint16_t* dout,
                                                     const uint16_t* pbuf,
                                                     const uint16_t* dsbuf, int L, int C,
                                                     uint16_t* dqkv) {
  __shared__ __attribute__((aligned(16))) uint16_t PT[QT * LMAX];   // [key][q]
  __shared__ __attribute__((aligned(16))) uint16_t ST[QT * LMAX];   // [key][q]
  __shared__ __attribute__((aligned(16))) uint16_t dOT[HD * LMAX];  // [d][q]
  __shared__ __attribute__((aligned(16))) uint16_t QTs[HD * LMAX];  // [d][q]
  const int kt = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int H = gridDim.y;
  const long row0 = (long)b * L;
  const long C3 = 3L * C;
  const long mat = ((long)b * H + h) * L * L;
  load_cols_t(PT, pbuf + mat, L, kt * QT);
  load_cols_t(ST, dsbuf + mat, L, kt * QT);
  load_rows_t(dOT, L, dout + row0 * C + h * HD, C, L);
  load_rows_t(QTs, L, qkv + row0 * C3 + h * HD, C3, L);
  __syncthreads();

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int m = lane & 15, g = lane >> 4;
  f32x4 dv[HD / 16], dk[HD / 16];
#pragma unroll
  for (int jd = 0; jd < HD / 16; ++jd) {
    dv[jd] = f32x4{0.f, 0.f, 0.f, 0.f};
    dk[jd] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  for (int ks = 0; ks < L / 32; ++ks) {
    const bf16x8 ap = ld8lds(PT + (w * 16 + m) * L + ks * 32 + g * 8);
    const bf16x8 as = ld8lds(ST + (w * 16 + m) * L + ks * 32 + g * 8);
#pragma unroll
    for (int jd = 0; jd < HD / 16; ++jd) {
      dv[jd] = mma(ap, ld8lds(dOT + (jd * 16 + m) * L + ks * 32 + g * 8), dv[jd]);
      dk[jd] = mma(as, ld8lds(QTs + (jd * 16 + m) * L + ks * 32 + g * 8), dk[jd]);
    }
  }
  const long k0 = row0 + (long)kt * QT + w * 16;
#pragma unroll
  for (int jd = 0; jd < HD / 16; ++jd)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const long r = (k0 + 4 * g + i) * C3 + h * HD + jd * 16 + m;
      dqkv[r + C] = bf(dk[jd][i]);
      dqkv[r + 2 * C] = bf(dv[jd][i]);
    }
}

}  // namespace

bool attn_fits(int L, int C, int heads) {
  return L >= QT && L % QT == 0 && L <= LMAX && C == heads * HD;
}

hipError_t launch_attn_fwd(const void* qkv, int B, int L, int C, int heads, void* o, void* pbuf,
                           hipStream_t st) {
  if (!attn_fits(L, C, heads)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_attn_fwd, dim3(L / QT, heads, B), dim3(256), 0, st,
                     static_cast<const uint16_t*>(qkv), L, C, static_cast<uint16_t*>(o),
                     static_cast<uint16_t*>(pbuf));
  return hipGetLastError();
}

hipError_t launch_attn_bwd(const void* qkv, const void* dout, const void* pbuf, int B, int L,
                           int C, int heads, void* dqkv, void* dsbuf, hipStream_t st) {
  if (!attn_fits(L, C, heads)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_attn_bwd_q, dim3(L / QT, heads, B), dim3(256), 0, st,
                     static_cast<const uint16_t*>(qkv), static_cast<const uint16_t*>(dout),
                     static_cast<const uint16_t*>(pbuf), L, C, static_cast<uint16_t*>(dqkv),
                     static_cast<uint16_t*>(dsbuf));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_attn_bwd_kv, dim3(L / QT, heads, B), dim3(256), 0, st,
                     static_cast<const uint16_t*>(qkv), static_cast<const uint16_t*>(dout),
                     static_cast<const uint16_t*>(pbuf), static_cast<const uint16_t*>(dsbuf), L,
                     C, static_cast<uint16_t*>(dqkv));
  return hipGetLastError();
}

}  // namespace pulse
