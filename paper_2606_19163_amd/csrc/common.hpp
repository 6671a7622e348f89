// Shared device-side types and helpers of the stage kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pulse {

enum DType : int { DT_F32 = 0, DT_BF16 = 1 };

// One NHWC tensor: element type and channel stride (the tensor's C).
struct Src {
  const void* ptr;
  int dtype;
  int C;
};

// A virtual NHWC input of C channels read from up to two tensors without
// materialising their concatenation: channel c < c0 comes from s0[c],
// channel c >= c0 from s1[c - c0].  `add` (fp32, C channels, may be null)
// is added element by element; it carries a buffered skip gradient into the
// gradient that reaches a cached encoder output.
struct VIn {
  Src s0, s1;
  int c0, C;
  const float* add;
};

struct Geo {
  int B, H, W;
  __host__ __device__ long pixels() const { return (long)B * H * W; }
  __host__ __device__ int hw() const { return H * W; }
};

// ---- bf16 helpers --------------------------------------------------------

__device__ __forceinline__ float bf2f(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

// fp32 -> bf16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint16_t f2bf(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

__device__ __forceinline__ uint32_t pack2(float a, float b) {
  typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;
  const bf16x2_t v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// Load 8 consecutive channels [c, c+8) of one pixel of a tensor as fp32.
__device__ __forceinline__ void ld8(const Src& s, long pix, int c, float v[8]) {
  if (s.dtype == DT_BF16) {
    const uint4 q = *reinterpret_cast<const uint4*>(
        static_cast<const uint16_t*>(s.ptr) + pix * s.C + c);
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  } else {
    const float4* p = reinterpret_cast<const float4*>(
        static_cast<const float*>(s.ptr) + pix * s.C + c);
    const float4 a = p[0], b = p[1];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
}

// Load channels [c, c+8) of pixel `pix` of a virtual input (c multiple of 8,
// the 8 channels never straddle the two sources because c0 % 8 == 0).
__device__ __forceinline__ void ld8v(const VIn& v, long pix, int c, float out[8]) {
  if (c < v.c0)
    ld8(v.s0, pix, c, out);
  else
    ld8(v.s1, pix, c - v.c0, out);
  if (v.add) {
    const float4* p = reinterpret_cast<const float4*>(v.add + pix * v.C + c);
    const float4 a = p[0], b = p[1];
    out[0] += a.x; out[1] += a.y; out[2] += a.z; out[3] += a.w;
    out[4] += b.x; out[5] += b.y; out[6] += b.z; out[7] += b.w;
  }
}

// Store 8 fp32 values as channels [c, c+8) of pixel `pix` of a tensor.
__device__ __forceinline__ void st8(void* ptr, int dtype, int C, long pix, int c,
                                    const float v[8]) {
  if (dtype == DT_BF16) {
    uint4 q;
    q.x = pack2(v[0], v[1]);
    q.y = pack2(v[2], v[3]);
    q.z = pack2(v[4], v[5]);
    q.w = pack2(v[6], v[7]);
    *reinterpret_cast<uint4*>(static_cast<uint16_t*>(ptr) + pix * C + c) = q;
  } else {
    float4* p = reinterpret_cast<float4*>(static_cast<float*>(ptr) + pix * C + c);
    p[0] = make_float4(v[0], v[1], v[2], v[3]);
    p[1] = make_float4(v[4], v[5], v[6], v[7]);
  }
}

// sigmoid(z) = 1 / (1 + e^-z) with the hardware reciprocal (v_rcp_f32,
// 1 ulp) in place of a correctly rounded division; e^-z overflowing to
// +inf gives exactly 0
__device__ __forceinline__ float sigmoid_f(float z) {
  return __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

__device__ __forceinline__ float silu_f(float z) { return z * sigmoid_f(z); }

// d SiLU(z)/dz
__device__ __forceinline__ float dsilu_f(float z) {
  const float s = sigmoid_f(z);
  return s * (1.0f + z * (1.0f - s));
}

// erf(x) by Abramowitz and Stegun, Handbook of Mathematical Functions,
// 7.1.26: erf(x) = 1 - t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) e^(-x^2)
// with t = 1 / (1 + p x) for x >= 0, odd in x; absolute error <= 1.5e-7,
// branch-free.  e2 = e^(-x^2) is passed in so that callers can share it.
__device__ __forceinline__ float erf_as(float x, float e2) {
  const float ax = fabsf(x);
  const float t = __builtin_amdgcn_rcpf(1.0f + 0.3275911f * ax);
  const float poly =
      t * (0.254829592f +
           t * (-0.284496736f + t * (1.421413741f + t * (-1.453152027f + t * 1.061405429f))));
  return copysignf(1.0f - poly * e2, x);
}

// GELU(z) = z * Phi(z) with the standard normal CDF Phi (erf form)
__device__ __forceinline__ float gelu_f(float z) {
  const float e2 = __expf(-0.5f * z * z);
  return 0.5f * z * (1.0f + erf_as(z * 0.70710678118654752f, e2));
}

// d GELU(z)/dz = Phi(z) + z * phi(z)
__device__ __forceinline__ float gelu_d(float z) {
  const float e2 = __expf(-0.5f * z * z);
  return 0.5f * (1.0f + erf_as(z * 0.70710678118654752f, e2)) + z * 0.39894228040143268f * e2;
}

}  // namespace pulse
