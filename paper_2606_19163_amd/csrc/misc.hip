// Timestep-embedding projection, weight re-layouts and conversions (gfx950).
// All small or streaming; none is on the MFMA path.
#include <algorithm>

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

// Every block's projection of one stage half in one launch.  Block
// (row tile, stage block k, image group) of 4 waves, each wave 2 rows o of
// Wl_k for 8 images.  Per slice of d every memory read is issued at once:
// the wave's Wl rows (16-byte loads into registers) and SiLU(temb) of the 8
// images (16-byte loads, activated into LDS); the lanes' 2 x 8 partial dot
// products then meet in LDS in a fixed order.  The blocks of the first row
// tile of stage block 0 also write the temb copy.
constexpr int TP_ROWS = 2;                      // rows per wave
constexpr int TP_IMG = 8;                       // images per block
constexpr int TP_DS = 2048;                     // d slice
constexpr int TP_J = TP_DS / 256;               // float4 loads per lane and row

__global__ __launch_bounds__(256) void k_temb_fwd_multi(const void* temb, int dtype, int B,
                                                        int D, TembFwdSet set, void* copy) {
  __shared__ __attribute__((aligned(16))) float st[TP_IMG][TP_DS];
  __shared__ float red[4][TP_ROWS * TP_IMG][65];
  const int k = blockIdx.y;
  const TembFwdBlock& blk = set.blk[k];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int b0 = blockIdx.z * TP_IMG;
  const int o0 = (blockIdx.x * 4 + wave) * TP_ROWS;
  const bool do_copy = copy && blockIdx.x == 0 && k == 0;
  const bool vec = dtype == DT_BF16 && (D % 8) == 0;
  float acc[TP_ROWS][TP_IMG];
#pragma unroll
  for (int r = 0; r < TP_ROWS; ++r)
#pragma unroll
    for (int i = 0; i < TP_IMG; ++i) acc[r][i] = 0.f;
  for (int dc = 0; dc < D; dc += TP_DS) {
    const int dn = min(TP_DS, D - dc);
    // the wave's weight rows, all loads in flight together
    float4 wv[TP_ROWS][TP_J];
#pragma unroll
    for (int r = 0; r < TP_ROWS; ++r) {
      const int o = min(o0 + r, blk.O - 1);
      const float* w = blk.Wl + (long)o * D + dc;
#pragma unroll
      for (int j = 0; j < TP_J; ++j) {
        const int d = 4 * lane + 256 * j;
        if ((D & 3) == 0 && d + 3 < dn) {
          wv[r][j] = *reinterpret_cast<const float4*>(w + d);
        } else {
          wv[r][j].x = d < dn ? w[d] : 0.f;
          wv[r][j].y = d + 1 < dn ? w[d + 1] : 0.f;
          wv[r][j].z = d + 2 < dn ? w[d + 2] : 0.f;
          wv[r][j].w = d + 3 < dn ? w[d + 3] : 0.f;
        }
      }
    }
    __syncthreads();  // the previous slice's LDS reads are done
    if (vec) {
      // 8-element pieces: TP_IMG * dn / 8 of them, at most 8 per thread
      constexpr int NP = TP_IMG * TP_DS / 8 / 256;
      uint4 q[NP];
#pragma unroll
      for (int j = 0; j < NP; ++j) {
        const int e = threadIdx.x + 256 * j;
        const int i = e / (TP_DS / 8), d = (e - i * (TP_DS / 8)) * 8;
        q[j] = uint4{0u, 0u, 0u, 0u};
        if (b0 + i < B && d < dn)
          q[j] = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(temb) +
                                                 (long)(b0 + i) * D + dc + d);
      }
#pragma unroll
      for (int j = 0; j < NP; ++j) {
        const int e = threadIdx.x + 256 * j;
        const int i = e / (TP_DS / 8), d = (e - i * (TP_DS / 8)) * 8;
        if (do_copy && b0 + i < B && d < dn)
          *reinterpret_cast<uint4*>(static_cast<uint16_t*>(copy) + (long)(b0 + i) * D + dc + d) =
              q[j];
        const uint32_t w4[4] = {q[j].x, q[j].y, q[j].z, q[j].w};
        float v[8];
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          v[2 * h] = silu_f(__uint_as_float(w4[h] << 16));
          v[2 * h + 1] = silu_f(__uint_as_float(w4[h] & 0xffff0000u));
        }
        if (!(b0 + i < B && d < dn)) {
#pragma unroll
          for (int h = 0; h < 8; ++h) v[h] = 0.f;
        }
        float4* dst = reinterpret_cast<float4*>(&st[i][d]);
        dst[0] = make_float4(v[0], v[1], v[2], v[3]);
        dst[1] = make_float4(v[4], v[5], v[6], v[7]);
      }
    } else {
      for (int e = threadIdx.x; e < TP_IMG * TP_DS; e += 256) {
        const int i = e / TP_DS, d = e - i * TP_DS;
        float v = 0.f;
        if (b0 + i < B && d < dn) {
          const long at = (long)(b0 + i) * D + dc + d;
          const float t = ld_any(temb, dtype, at);
          if (do_copy) st_any(copy, dtype, at, t);
          v = silu_f(t);
        }
        st[i][d] = v;
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < TP_J; ++j) {
      const int d = 4 * lane + 256 * j;
      if (d >= dn) break;
#pragma unroll
      for (int i = 0; i < TP_IMG; ++i) {
        const float4 sv = *reinterpret_cast<const float4*>(&st[i][d]);
#pragma unroll
        for (int r = 0; r < TP_ROWS; ++r)
          acc[r][i] += wv[r][j].x * sv.x + wv[r][j].y * sv.y + wv[r][j].z * sv.z +
                       wv[r][j].w * sv.w;
      }
    }
  }
  // lane sums -> LDS; lane q < 16 of the wave then adds the 64 lanes of
  // (row q / 8, image q % 8) in order
#pragma unroll
  for (int r = 0; r < TP_ROWS; ++r)
#pragma unroll
    for (int i = 0; i < TP_IMG; ++i) red[wave][r * TP_IMG + i][lane] = acc[r][i];
  __syncthreads();
  if (lane < TP_ROWS * TP_IMG) {
    const int r = lane / TP_IMG, i = lane - r * TP_IMG;
    const int o = o0 + r, b = b0 + i;
    if (o < blk.O && b < B) {
      float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
      for (int l = 0; l < 64; l += 4) {
        s0 += red[wave][lane][l];
        s1 += red[wave][lane][l + 1];
        s2 += red[wave][lane][l + 2];
        s3 += red[wave][lane][l + 3];
      }
      float bias = blk.bias_a[o];
      if (blk.bias_b) bias += blk.bias_b[o];
      blk.e[(long)b * blk.ldE + o] = ((s0 + s1) + (s2 + s3)) + bias;
    }
  }
}

// dWl[o][d] += sum_b de[b][o] * SiLU(temb[b][d]) over a 64 (d) x 16 (o)
// tile per block: the tile's SiLU(temb) columns and de rows are staged in
// LDS for up to 32 images at a time (each SiLU evaluated once per tile, not
// once per output), and thread (d lane, row group g) owns rows 4 g .. 4 g + 3.
// The blocks of the first d tile also sum de over the images for the bias
// gradients.  Every sum runs over b in increasing order.
constexpr int TB_D = 64, TB_O = 16, TB_B = 32;
__global__ __launch_bounds__(256) void k_temb_bwd_w(const float* de, const void* temb, int dtype,
                                                    int B, int D, int O, float* dWl, float* dbl,
                                                    float* db1) {
  __shared__ float sv[TB_B][TB_D];
  __shared__ __attribute__((aligned(16))) float se[TB_B][TB_O];
  const int tx = threadIdx.x & 63, g = threadIdx.x >> 6;
  const int d0 = blockIdx.x * TB_D, o0 = blockIdx.y * TB_O;
  const bool bias = blockIdx.x == 0 && threadIdx.x < TB_O;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  float sb = 0.f;
  for (int b0 = 0; b0 < B; b0 += TB_B) {
    const int nb = min(TB_B, B - b0);
    __syncthreads();
    for (int e = threadIdx.x; e < nb * TB_D; e += 256) {
      const int bb = e / TB_D, c = e - bb * TB_D;
      sv[bb][c] = d0 + c < D ? silu_f(ld_any(temb, dtype, (long)(b0 + bb) * D + d0 + c)) : 0.f;
    }
    for (int e = threadIdx.x; e < nb * TB_O; e += 256) {
      const int bb = e / TB_O, c = e - bb * TB_O;
      se[bb][c] = o0 + c < O ? de[(long)(b0 + bb) * O + o0 + c] : 0.f;
    }
    __syncthreads();
    for (int bb = 0; bb < nb; ++bb) {
      const float v = sv[bb][tx];
      const float4 w = reinterpret_cast<const float4*>(&se[bb][0])[g];
      acc[0] += w.x * v;
      acc[1] += w.y * v;
      acc[2] += w.z * v;
      acc[3] += w.w * v;
    }
    if (bias)
      for (int bb = 0; bb < nb; ++bb) sb += se[bb][threadIdx.x];
  }
  const int d = d0 + tx;
  if (d < D) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int o = o0 + 4 * g + j;
      if (o < O) dWl[(long)o * D + d] += acc[j];
    }
  }
  if (bias && o0 + threadIdx.x < O) {
    dbl[o0 + threadIdx.x] += sb;
    if (db1) db1[o0 + threadIdx.x] += sb;
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

hipError_t launch_temb_fwd_multi(const void* temb, int dtype, int B, int D,
                                 const TembFwdSet& set, void* copy, hipStream_t st) {
  if (set.n < 1 || set.n > TEMB_MAX_BLOCKS) return hipErrorInvalidValue;
  int omax = 0;
  for (int k = 0; k < set.n; ++k) omax = std::max(omax, set.blk[k].O);
  const int rows_per_block = 4 * TP_ROWS;
  hipLaunchKernelGGL(k_temb_fwd_multi,
                     dim3((omax + rows_per_block - 1) / rows_per_block, set.n,
                          (B + TP_IMG - 1) / TP_IMG),
                     dim3(256), 0, st, temb, dtype, B, D, set, copy);
  return hipGetLastError();
}

hipError_t launch_temb_bwd(const float* de, const void* temb, int dtype, int B, int D, int O,
                           const float* Wl, float* dWl, float* dbl, float* db1, float* dtemb,
                           hipStream_t st) {
  if (O <= 0) return hipSuccess;
  // at least one d tile: its blocks also produce the bias gradients
  const int dt = std::max(1, (D + TB_D - 1) / TB_D);
  hipLaunchKernelGGL(k_temb_bwd_w, dim3(dt, (O + TB_O - 1) / TB_O), dim3(256), 0, st, de, temb,
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
