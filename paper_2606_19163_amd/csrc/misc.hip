// Timestep-embedding projection, weight re-layouts and conversions (gfx950).
// All small or streaming; none is on the MFMA path.
#include "common.hpp"
#include "kernels.hpp"

namespace pulse {

namespace {

__device__ __forceinline__ float ld_any(const void* p, int dtype, long i) {
  return dtype == DT_BF16 ? bf2f(static_cast<const uint16_t*>(p)[i])
                          : static_cast<const float*>(p)[i];
}

__device__ __forceinline__ void st_any(void* p, int dtype, long i, float v) {
  if (dtype == DT_BF16)
    static_cast<uint16_t*>(p)[i] = f2bf(v);
  else
    static_cast<float*>(p)[i] = v;
}

// one wave per (o, b): lanes stride over d (four loads in flight per lane),
// xor-shuffle tree reduction
__global__ __launch_bounds__(64) void k_temb_fwd(const void* temb, int dtype, int D, int O,
                                                 const float* Wl, const float* bias_a,
                                                 const float* bias_b, float* e) {
  const int o = blockIdx.x, b = blockIdx.y;
  const float* w = Wl + (long)o * D;
  const long t0 = (long)b * D;
  float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
  int d = threadIdx.x;
  for (; d + 192 < D; d += 256) {
    const float w0 = w[d], w1 = w[d + 64], w2 = w[d + 128], w3 = w[d + 192];
    const float x0 = ld_any(temb, dtype, t0 + d), x1 = ld_any(temb, dtype, t0 + d + 64);
    const float x2 = ld_any(temb, dtype, t0 + d + 128), x3 = ld_any(temb, dtype, t0 + d + 192);
    s0 += w0 * silu_f(x0);
    s1 += w1 * silu_f(x1);
    s2 += w2 * silu_f(x2);
    s3 += w3 * silu_f(x3);
  }
  for (; d < D; d += 64) s0 += w[d] * silu_f(ld_any(temb, dtype, t0 + d));
  float s = (s0 + s1) + (s2 + s3);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if (threadIdx.x == 0) {
    float bias = bias_a[o];
    if (bias_b) bias += bias_b[o];
    e[(long)b * O + o] = s + bias;
  }
}

// thread (o, d): dWl[o][d] += sum_b de[b][o] * SiLU(temb[b][d]); the extra
// thread d == D of each row accumulates the bias gradients.
__global__ void k_temb_bwd_w(const float* de, const void* temb, int dtype, int B, int D, int O,
                             float* dWl, float* dbl, float* db1) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long)O * (D + 1)) return;
  const int o = (int)(i / (D + 1));
  const int d = (int)(i - (long)o * (D + 1));
  if (d < D) {
    float s = 0.f;
    for (int b = 0; b < B; ++b)
      s += de[(long)b * O + o] * silu_f(ld_any(temb, dtype, (long)b * D + d));
    dWl[(long)o * D + d] += s;
  } else {
    float s = 0.f;
    for (int b = 0; b < B; ++b) s += de[(long)b * O + o];
    dbl[o] += s;
    if (db1) db1[o] += s;
  }
}

// block (64 d x 16 o-lanes) per (d block, image b):
// dtemb[b][d] += SiLU'(temb[b][d]) * sum_o Wl[o][d] de[b][o]
__global__ __launch_bounds__(1024) void k_temb_bwd_x(const float* de, const void* temb,
                                                     int dtype, int B, int D, int O,
                                                     const float* Wl, float* dtemb) {
  __shared__ float sm[16][64];
  const int d = blockIdx.x * 64 + threadIdx.x;
  const int b = blockIdx.y;
  float s = 0.f;
  if (d < D) {
    int o = threadIdx.y;
    for (; o + 48 < O; o += 64) {
      const float w0 = Wl[(long)o * D + d], w1 = Wl[(long)(o + 16) * D + d];
      const float w2 = Wl[(long)(o + 32) * D + d], w3 = Wl[(long)(o + 48) * D + d];
      s += w0 * de[(long)b * O + o];
      s += w1 * de[(long)b * O + o + 16];
      s += w2 * de[(long)b * O + o + 32];
      s += w3 * de[(long)b * O + o + 48];
    }
    for (; o < O; o += 16) s += Wl[(long)o * D + d] * de[(long)b * O + o];
  }
  sm[threadIdx.y][threadIdx.x] = s;
  __syncthreads();
  if (threadIdx.y == 0 && d < D) {
    float t = sm[0][threadIdx.x];
#pragma unroll
    for (int y = 1; y < 16; ++y) t += sm[y][threadIdx.x];
    const long i = (long)b * D + d;
    dtemb[i] += t * dsilu_f(ld_any(temb, dtype, i));
  }
}

__global__ void k_convert_rows(const float* src, int rows, int cols, void* dst, int ldd,
                               int col_off, int dtype) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long)rows * cols) return;
  const long r = i / cols;
  const long c = i - r * cols;
  st_any(dst, dtype, r * ldd + col_off + c, src[i]);
}

__global__ void k_flip3x3(const float* src, int O, int C, void* dst, int dtype) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long)O * 9 * C) return;
  // destination index (c, t, o)
  const int o = (int)(i % O);
  const long ct = i / O;
  const int t = (int)(ct % 9);
  const int c = (int)(ct / 9);
  st_any(dst, dtype, i, src[((long)o * 9 + (8 - t)) * C + c]);
}

__global__ void k_transpose(const float* src, int O, int C, void* dst, int dtype) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long)O * C) return;
  const int o = (int)(i % O);
  const int c = (int)(i / O);
  st_any(dst, dtype, i, src[(long)o * C + c]);
}

__global__ void k_vec_add(const float* a, const float* b, float* dst, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = a[i] + (b ? b[i] : 0.f);
}

__global__ void k_cast(const void* src, int sdt, void* dst, int ddt, long n) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (long)gridDim.x * blockDim.x)
    st_any(dst, ddt, i, ld_any(src, sdt, i));
}

// dst = (ddt) (a + b), a of dtype adt, b fp32
__global__ void k_add_cast(const void* a, int adt, const float* b, void* dst, int ddt, long n) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (long)gridDim.x * blockDim.x)
    st_any(dst, ddt, i, ld_any(a, adt, i) + b[i]);
}

// dst = a + b over n = 8 * n8 elements, 8 per thread per step (16- or
// 32-byte accesses); the element types are template arguments
template <int ADT, int DDT>
__global__ __launch_bounds__(256) void k_add_cast8(const void* a, const float* b, void* dst,
                                                   long n8) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n8;
       i += (long)gridDim.x * blockDim.x) {
    float v[8];
    ld8(Src{a, ADT, 8}, i, 0, v);
    const float4* q = reinterpret_cast<const float4*>(b) + 2 * i;
    const float4 b0 = q[0], b1 = q[1];
    v[0] += b0.x; v[1] += b0.y; v[2] += b0.z; v[3] += b0.w;
    v[4] += b1.x; v[5] += b1.y; v[6] += b1.z; v[7] += b1.w;
    st8(dst, DDT, 8, i, 0, v);
  }
}

unsigned nblk(long n, int t = 256) { return (unsigned)((n + t - 1) / t); }

}  // namespace

hipError_t launch_temb_fwd(const void* temb, int dtype, int B, int D, int O, const float* Wl,
                           const float* bias_a, const float* bias_b, float* e,
                           hipStream_t st) {
  hipLaunchKernelGGL(k_temb_fwd, dim3(O, B), dim3(64), 0, st, temb, dtype, D, O, Wl, bias_a,
                     bias_b, e);
  return hipGetLastError();
}

hipError_t launch_temb_bwd(const float* de, const void* temb, int dtype, int B, int D, int O,
                           const float* Wl, float* dWl, float* dbl, float* db1, float* dtemb,
                           hipStream_t st) {
  hipLaunchKernelGGL(k_temb_bwd_w, dim3(nblk((long)O * (D + 1))), dim3(256), 0, st, de, temb,
                     dtype, B, D, O, dWl, dbl, db1);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !dtemb) return e;
  hipLaunchKernelGGL(k_temb_bwd_x, dim3((D + 63) / 64, B), dim3(64, 16), 0, st, de, temb, dtype,
                     B, D, O, Wl, dtemb);
  return hipGetLastError();
}

hipError_t launch_convert_rows(const float* src, int rows, int cols, void* dst, int ldd,
                               int col_off, int dtype, hipStream_t st) {
  hipLaunchKernelGGL(k_convert_rows, dim3(nblk((long)rows * cols)), dim3(256), 0, st, src, rows,
                     cols, dst, ldd, col_off, dtype);
  return hipGetLastError();
}

hipError_t launch_flip3x3(const float* src, int O, int C, void* dst, int dtype,
                          hipStream_t st) {
  hipLaunchKernelGGL(k_flip3x3, dim3(nblk((long)O * 9 * C)), dim3(256), 0, st, src, O, C, dst,
                     dtype);
  return hipGetLastError();
}

hipError_t launch_transpose(const float* src, int O, int C, void* dst, int dtype,
                            hipStream_t st) {
  hipLaunchKernelGGL(k_transpose, dim3(nblk((long)O * C)), dim3(256), 0, st, src, O, C, dst,
                     dtype);
  return hipGetLastError();
}

hipError_t launch_vec_add(const float* a, const float* b, float* dst, int n, hipStream_t st) {
  hipLaunchKernelGGL(k_vec_add, dim3(nblk(n)), dim3(256), 0, st, a, b, dst, n);
  return hipGetLastError();
}

hipError_t launch_cast(const void* src, int sdt, void* dst, int ddt, long n, hipStream_t st) {
  long b = (n + 255) / 256;
  if (b > 8192) b = 8192;
  if (b < 1) b = 1;
  hipLaunchKernelGGL(k_cast, dim3((unsigned)b), dim3(256), 0, st, src, sdt, dst, ddt, n);
  return hipGetLastError();
}

hipError_t launch_add_cast(const void* a, int adt, const float* b, void* dst, int ddt, long n,
                           hipStream_t st) {
  const bool aligned = ((reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(b) |
                         reinterpret_cast<uintptr_t>(dst)) & 15) == 0;
  if (n % 8 == 0 && aligned) {
    long blocks = (n / 8 + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    if (blocks < 1) blocks = 1;
    auto kern = adt == DT_BF16 ? (ddt == DT_BF16 ? k_add_cast8<DT_BF16, DT_BF16>
                                                 : k_add_cast8<DT_BF16, DT_F32>)
                               : (ddt == DT_BF16 ? k_add_cast8<DT_F32, DT_BF16>
                                                 : k_add_cast8<DT_F32, DT_F32>);
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(256), 0, st, a, b, dst, n / 8);
    return hipGetLastError();
  }
  long blocks = (n + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_add_cast, dim3((unsigned)blocks), dim3(256), 0, st, a, adt, b, dst, ddt,
                     n);
  return hipGetLastError();
}

}  // namespace pulse
