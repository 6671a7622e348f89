// LayerNorm and GELU of the transformer-block stage (gfx950): token-major
// [T][C] bf16 activations; one wave per token for the LayerNorm, each lane
// holding whole 8-channel vectors in registers; statistics in fp32.
#include <hip/hip_runtime.h>

#include "common.hpp"
#include "tkernels.hpp"

namespace pulse {

namespace {

constexpr int LN_VEC = 4;        // 8-channel vectors per lane: C <= 64 * 8 * LN_VEC = 2048
constexpr int LN_TOK = 1;        // tokens per wave in the backward pass

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ void ld8bf(const uint16_t* p, float v[8]) {
  const uint4 q = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

__device__ __forceinline__ void st8bf(uint16_t* p, const float v[8]) {
  uint4 q;
  q.x = pack2(v[0], v[1]);
  q.y = pack2(v[2], v[3]);
  q.z = pack2(v[4], v[5]);
  q.w = pack2(v[6], v[7]);
  *reinterpret_cast<uint4*>(p) = q;
}

// y = (x - mean) * rstd * g + b per token; stats[t] = (mean, rstd)
__global__ __launch_bounds__(256) void k_ln_fwd(const uint16_t* x, long T, int C, float eps,
                                                const float* g, const float* b, uint16_t* y,
                                                float2* stats) {
  const long t = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= T) return;
  const int nv = C / 8;
  float v[LN_VEC][8];
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < LN_VEC; ++j) {
    const int vi = lane + 64 * j;
    if (vi < nv) {
      ld8bf(x + t * C + vi * 8, v[j]);
#pragma unroll
      for (int i = 0; i < 8; ++i) s += v[j][i];
    }
  }
  const float mean = wave_sum(s) / C;
  float q = 0.f;
#pragma unroll
  for (int j = 0; j < LN_VEC; ++j)
    if (lane + 64 * j < nv)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float d = v[j][i] - mean;
        q += d * d;
      }
  const float rstd = rsqrtf(wave_sum(q) / C + eps);
#pragma unroll
  for (int j = 0; j < LN_VEC; ++j) {
    const int vi = lane + 64 * j;
    if (vi < nv) {
      float o[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] = (v[j][i] - mean) * rstd * g[vi * 8 + i] + b[vi * 8 + i];
      st8bf(y + t * C + vi * 8, o);
    }
  }
  if (lane == 0) stats[t] = make_float2(mean, rstd);
}

// dx = add + rstd * (dxh - mean(dxh) - xh * mean(dxh * xh)), dxh = dy * g;
// per-block partial sums of dy * xh (row 0) and dy (row 1) over the block's
// tokens go to part[block][2][C]
__global__ __launch_bounds__(256) void k_ln_bwd(const uint16_t* dy, const uint16_t* x,
                                                const float2* stats, const float* g,
                                                const uint16_t* add, long T, int C, uint16_t* dx,
                                                float* part, float* csum) {
  // per wave, [2][C / 4 per j] reused below; the partial-sum passes write
  // lanes * 8 values per row whatever LN_VEC is
  static_assert(64 * LN_VEC * 8 / 4 >= 64 * 8, "k_ln_bwd: LDS rows hold 64 lanes x 8 values");
  __shared__ float sm[4][2][64 * LN_VEC * 8 / 4];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nv = C / 8;
  float accg[LN_VEC][8], accb[LN_VEC][8], accx[LN_VEC][8];
#pragma unroll
  for (int j = 0; j < LN_VEC; ++j)
#pragma unroll
    for (int i = 0; i < 8; ++i) accg[j][i] = accb[j][i] = accx[j][i] = 0.f;
  for (int k = 0; k < LN_TOK; ++k) {
    const long t = ((long)blockIdx.x * 4 + w) * LN_TOK + k;
    if (t >= T) break;
    const float2 st = stats[t];
    float xh[LN_VEC][8], gy[LN_VEC][8];
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int j = 0; j < LN_VEC; ++j) {
      const int vi = lane + 64 * j;
      if (vi < nv) {
        float xv[8], dv[8];
        ld8bf(x + t * C + vi * 8, xv);
        ld8bf(dy + t * C + vi * 8, dv);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          xh[j][i] = (xv[i] - st.x) * st.y;
          gy[j][i] = dv[i] * g[vi * 8 + i];
          s1 += gy[j][i];
          s2 += gy[j][i] * xh[j][i];
          accg[j][i] += dv[i] * xh[j][i];
          accb[j][i] += dv[i];
        }
      }
    }
    const float m1 = wave_sum(s1) / C, m2 = wave_sum(s2) / C;
#pragma unroll
    for (int j = 0; j < LN_VEC; ++j) {
      const int vi = lane + 64 * j;
      if (vi < nv) {
        float o[8], a[8];
        if (add) {
          ld8bf(add + t * C + vi * 8, a);
        } else {
#pragma unroll
          for (int i = 0; i < 8; ++i) a[i] = 0.f;
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          o[i] = a[i] + st.y * (gy[j][i] - m1 - xh[j][i] * m2);
          accx[j][i] += bf2f(f2bf(o[i]));  // the value as stored
        }
        st8bf(dx + t * C + vi * 8, o);
      }
    }
  }
  // the four waves' channel sums, in wave order, one vector slice at a time
  float* out = part + (long)blockIdx.x * 2 * C;
#pragma unroll
  for (int j = 0; j < LN_VEC; ++j) {
    const int vi = lane + 64 * j;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      sm[w][0][lane * 8 + i] = accg[j][i];
      sm[w][1][lane * 8 + i] = accb[j][i];
    }
    __syncthreads();
    if (w == 0 && vi < nv) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        float sg = 0.f, sb = 0.f;
#pragma unroll
        for (int ww = 0; ww < 4; ++ww) {
          sg += sm[ww][0][lane * 8 + i];
          sb += sm[ww][1][lane * 8 + i];
        }
        out[vi * 8 + i] = sg;
        out[C + vi * 8 + i] = sb;
      }
    }
  }
  if (!csum) return;
  // column sums of dx as stored, to csum[block][0][C]
  float* cs = csum + (long)blockIdx.x * 2 * C;
#pragma unroll
  for (int j = 0; j < LN_VEC; ++j) {
    const int vi = lane + 64 * j;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 8; ++i) sm[w][0][lane * 8 + i] = accx[j][i];
    __syncthreads();
    if (w == 0 && vi < nv) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        float sx = 0.f;
#pragma unroll
        for (int ww = 0; ww < 4; ++ww) sx += sm[ww][0][lane * 8 + i];
        cs[vi * 8 + i] = sx;
      }
    }
  }
}


__global__ __launch_bounds__(256) void k_gelu_fwd(const uint16_t* z, uint16_t* m, long n8) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n8;
       i += (long)gridDim.x * blockDim.x) {
    float v[8];
    ld8bf(z + i * 8, v);
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = gelu_f(v[k]);
    st8bf(m + i * 8, v);
  }
}

__global__ __launch_bounds__(256) void k_gelu_bwd(const uint16_t* dm, const uint16_t* z,
                                                  uint16_t* dz, long n8) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n8;
       i += (long)gridDim.x * blockDim.x) {
    float a[8], v[8];
    ld8bf(dm + i * 8, a);
    ld8bf(z + i * 8, v);
#pragma unroll
    for (int k = 0; k < 8; ++k) a[k] *= gelu_d(v[k]);
    st8bf(dz + i * 8, a);
  }
}

unsigned grid_of(long n, long cap = 8192) {
  long b = (n + 255) / 256;
  return (unsigned)(b < 1 ? 1 : (b > cap ? cap : b));
}

}  // namespace

int ln_bwd_blocks(long T) { return (int)((T + 4 * LN_TOK - 1) / (4 * LN_TOK)); }

hipError_t launch_ln_fwd(const void* x, long T, int C, float eps, const float* g, const float* b,
                         void* y, float* stats, hipStream_t st) {
  if (C % 8 || C > 64 * 8 * LN_VEC) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_ln_fwd, dim3((unsigned)((T + 3) / 4)), dim3(256), 0, st,
                     static_cast<const uint16_t*>(x), T, C, eps, g, b, static_cast<uint16_t*>(y),
                     reinterpret_cast<float2*>(stats));
  return hipGetLastError();
}

hipError_t launch_ln_bwd(const void* dy, const void* x, const float* stats, const float* g,
                         const void* add, long T, int C, void* dx, float* part, float* csum,
                         hipStream_t st) {
  if (C % 8 || C > 64 * 8 * LN_VEC) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_ln_bwd, dim3((unsigned)ln_bwd_blocks(T)), dim3(256), 0, st,
                     static_cast<const uint16_t*>(dy), static_cast<const uint16_t*>(x),
                     reinterpret_cast<const float2*>(stats), g, static_cast<const uint16_t*>(add),
                     T, C, static_cast<uint16_t*>(dx), part, csum);
  return hipGetLastError();
}

hipError_t launch_gelu_fwd(const void* z, void* m, long n, hipStream_t st) {
  if (n % 8) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_gelu_fwd, dim3(grid_of(n / 8)), dim3(256), 0, st,
                     static_cast<const uint16_t*>(z), static_cast<uint16_t*>(m), n / 8);
  return hipGetLastError();
}


hipError_t launch_gelu_bwd(const void* dm, const void* z, void* dz, long n, hipStream_t st) {
  if (n % 8) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_gelu_bwd, dim3(grid_of(n / 8)), dim3(256), 0, st,
                     static_cast<const uint16_t*>(dm), static_cast<const uint16_t*>(z),
                     static_cast<uint16_t*>(dz), n / 8);
  return hipGetLastError();
}

}  // namespace pulse
