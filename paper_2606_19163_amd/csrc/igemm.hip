// Implicit-GEMM convolution on CDNA4 (gfx950) matrix cores.
//
// One kernel template serves the three contractions of a stride-1 3x3 / 1x1
// conv over NHWC activations:
//
//  * CONV mode (forward and data gradient): C[m, n] = sum_k A[m, k] B[n, k]
//    with m a pixel, n an output channel and k = (segment, tap, channel).
//    A is never materialised: a K-step of BK columns lies inside one tap of
//    one segment, so the block copies BK consecutive channels of the pixel
//    shifted by that tap (zero outside the image) straight from the NHWC
//    source(s).  A segment is a 3x3 or 1x1 conv over a virtual input that
//    may read two tensors (the decoder's [upstream || skip]); several
//    segments side by side along K fuse the 1x1 shortcut into the second
//    3x3 conv of a block.  B is a row-major [N][K] weight matrix (for the
//    data gradient: the flipped, transposed 3x3 weights).  The epilogue adds
//    bias / per-image row vector / residual and writes whole 16-byte vectors
//    from an LDS-staged tile.
//  * WGRAD mode (weight gradient): C[m, n] = sum_p dY[p, m] X[p + tap(n),
//    c(n)] with m an output channel, n = (segment, tap, channel) and the
//    contraction over pixels p, split across blockIdx.z into fixed pixel
//    ranges whose fp32 partials a finalize kernel sums in a fixed order.
//    Both operands are pixel-strided in NHWC, so each thread copies an 8x8
//    (pixel x channel) micro-tile and transposes it in registers (byte
//    permutes) before the LDS store.
//
// Operands are copied raw in the compute dtype (every conversion happens in
// the memory-bound kernels that produce them).  bf16 operands use
// v_mfma_f32_16x16x32_bf16 with fp32 accumulation; the fp32 path uses
// v_mfma_f32_16x16x4_f32.  Operand tiles are staged in LDS (K-contiguous rows
// padded against bank conflicts), double buffered, with the next tile's
// global loads in flight while the current one is consumed.
#include "common.hpp"
#include "kernels.hpp"

namespace pulse {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

template <int BM_, int BN_, int BK_, int WM_, int WN_, bool F32_>
struct Cfg {
  static constexpr int BM = BM_, BN = BN_, BK = BK_, WM = WM_, WN = WN_;
  static constexpr bool F32 = F32_;
  static constexpr int WAVES_M = BM / WM, WAVES_N = BN / WN;
  static constexpr int NT = WAVES_M * WAVES_N * 64;
  static constexpr int TM = WM / 16, TN = WN / 16;
  static constexpr int ESZ = F32 ? 4 : 2;         // bytes per element
  static constexpr int LDK = BK + (F32 ? 4 : 8);  // padded LDS row (elements)
  static constexpr int KV = BK / 8;               // 8-element vectors per row
  static constexpr int VW = F32 ? 8 : 4;          // 32-bit words per vector
  static constexpr int LDS_A = BM * LDK * ESZ;
  static constexpr int LDS_B = BN * LDK * ESZ;
  static constexpr int LDS_OPS = 2 * (LDS_A + LDS_B);
  static constexpr int LDC = BN + 4;              // fp32 epilogue tile row
  static constexpr int LDS_EPI = BM * LDC * 4;
  static constexpr int LDS_BYTES = LDS_OPS > LDS_EPI ? LDS_OPS : LDS_EPI;
  // CONV mode: vectors per thread for the A and B tiles
  static constexpr int NVA = (BM * KV) / NT;
  static constexpr int NVB = (BN * KV) / NT;
  // WGRAD mode: 8x8 micro-tiles per thread
  static constexpr int NMA = (BM / 8) * (BK / 8);
  static constexpr int NMB = (BN / 8) * (BK / 8);
  static constexpr int NMT = (NMA + NMB + NT - 1) / NT;
  static_assert(BM % WM == 0 && BN % WN == 0 && WM % 16 == 0 && WN % 16 == 0, "tile");
  static_assert(BK % 32 == 0, "BK");
  static_assert((BM * KV) % NT == 0 && (BN * KV) % NT == 0, "vector split");
  static_assert(LDS_BYTES <= 160 * 1024, "LDS");
};

// 8 operand elements: 8 fp32 words or 4 words of bf16 pairs
template <bool F32>
struct VecT {
  uint32_t w[F32 ? 8 : 4];
};

template <bool F32>
__device__ __forceinline__ void vzero(VecT<F32>& v) {
#pragma unroll
  for (int i = 0; i < (F32 ? 8 : 4); ++i) v.w[i] = 0u;
}

// Raw copy of 8 elements of the compute dtype.
template <bool F32>
__device__ __forceinline__ void vload(const void* p, VecT<F32>& v) {
  const uint4 q0 = reinterpret_cast<const uint4*>(p)[0];
  v.w[0] = q0.x; v.w[1] = q0.y; v.w[2] = q0.z; v.w[3] = q0.w;
  if constexpr (F32) {
    const uint4 q1 = reinterpret_cast<const uint4*>(p)[1];
    v.w[F32 ? 4 : 0] = q1.x; v.w[F32 ? 5 : 1] = q1.y;
    v.w[F32 ? 6 : 2] = q1.z; v.w[F32 ? 7 : 3] = q1.w;
  }
}

template <class C>
__device__ __forceinline__ void lds_put(char* base, int row, int k, const VecT<C::F32>& v) {
  char* p = base + (row * C::LDK + k) * C::ESZ;
  reinterpret_cast<uint4*>(p)[0] = make_uint4(v.w[0], v.w[1], v.w[2], v.w[3]);
  if constexpr (C::F32)
    reinterpret_cast<uint4*>(p)[1] = make_uint4(v.w[C::F32 ? 4 : 0], v.w[C::F32 ? 5 : 1],
                                                v.w[C::F32 ? 6 : 2], v.w[C::F32 ? 7 : 3]);
}

// Address of channel c of pixel pix of a raw two-source input.
template <bool F32>
__device__ __forceinline__ const char* vaddr(const VIn& v, long pix, int c) {
  constexpr int esz = F32 ? 4 : 2;
  if (c < v.c0) return static_cast<const char*>(v.s0.ptr) + (pix * v.s0.C + c) * esz;
  return static_cast<const char*>(v.s1.ptr) + (pix * v.s1.C + (c - v.c0)) * esz;
}

// Transpose an 8x8 block: in[e] holds 8 channels of pixel e, out[q] gets 8
// pixels of channel q.
template <bool F32>
__device__ __forceinline__ void transpose8(const VecT<F32> (&in)[8], VecT<F32> (&out)[8]) {
  if constexpr (F32) {
#pragma unroll
    for (int q = 0; q < 8; ++q)
#pragma unroll
      for (int e = 0; e < 8; ++e) out[q].w[e] = in[e].w[q];
  } else {
    // out[q].w[j] = (channel q of pixel 2j) | (channel q of pixel 2j+1) << 16
#pragma unroll
    for (int q = 0; q < 8; ++q)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t lo = in[2 * j].w[q / 2], hi = in[2 * j + 1].w[q / 2];
        out[q].w[j] = (q & 1) ? __builtin_amdgcn_perm(hi, lo, 0x07060302u)
                              : __builtin_amdgcn_perm(hi, lo, 0x05040100u);
      }
  }
}

// Which segment holds index `i` (segments are sorted and contiguous).
__device__ __forceinline__ int seg_of(int nseg, int b1, int b2, int i) {
  int s = 0;
  if (nseg > 1 && i >= b1) s = 1;
  if (nseg > 2 && i >= b2) s = 2;
  return s;
}

// Remap the linear block id so that consecutive tiles land on one XCD
// (the hardware deals workgroups round-robin over the 8 XCDs).
__device__ __forceinline__ int xcd_remap(int bid, int nb) {
  if (nb % 8 != 0) return bid;
  return (bid % 8) * (nb / 8) + bid / 8;
}

template <class C>
__device__ __forceinline__ void mma_tile(const char* As, const char* Bs, int wm, int wn,
                                         int lane, f32x4_t (&acc)[C::TM][C::TN]) {
  const int r16 = lane & 15;
  const int kq = (lane >> 4) * 8;
#pragma unroll
  for (int s = 0; s < C::BK / 32; ++s) {
    const int k = s * 32 + kq;
    if constexpr (C::F32) {
      float af[C::TM][8], bfr[C::TN][8];
#pragma unroll
      for (int i = 0; i < C::TM; ++i) {
        const float* p = reinterpret_cast<const float*>(As) +
                         (wm * C::WM + i * 16 + r16) * C::LDK + k;
        const float4 x0 = reinterpret_cast<const float4*>(p)[0];
        const float4 x1 = reinterpret_cast<const float4*>(p)[1];
        af[i][0] = x0.x; af[i][1] = x0.y; af[i][2] = x0.z; af[i][3] = x0.w;
        af[i][4] = x1.x; af[i][5] = x1.y; af[i][6] = x1.z; af[i][7] = x1.w;
      }
#pragma unroll
      for (int j = 0; j < C::TN; ++j) {
        const float* p = reinterpret_cast<const float*>(Bs) +
                         (wn * C::WN + j * 16 + r16) * C::LDK + k;
        const float4 x0 = reinterpret_cast<const float4*>(p)[0];
        const float4 x1 = reinterpret_cast<const float4*>(p)[1];
        bfr[j][0] = x0.x; bfr[j][1] = x0.y; bfr[j][2] = x0.z; bfr[j][3] = x0.w;
        bfr[j][4] = x1.x; bfr[j][5] = x1.y; bfr[j][6] = x1.z; bfr[j][7] = x1.w;
      }
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
#pragma unroll
          for (int e = 0; e < 8; ++e)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i][e], bfr[j][e],
                                                             acc[i][j], 0, 0, 0);
    } else {
      bf16x8_t af[C::TM], bfr[C::TN];
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
        af[i] = *reinterpret_cast<const bf16x8_t*>(
            As + ((wm * C::WM + i * 16 + r16) * C::LDK + k) * 2);
#pragma unroll
      for (int j = 0; j < C::TN; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8_t*>(
            Bs + ((wn * C::WN + j * 16 + r16) * C::LDK + k) * 2);
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j],
                                                              0, 0, 0);
    }
  }
}

// Park the accumulators of every wave in an fp32 [BM][LDC] LDS tile.
template <class C>
__device__ __forceinline__ void acc_to_lds(float* ct, int wm, int wn, int lane,
                                           const f32x4_t (&acc)[C::TM][C::TN]) {
  const int r16 = lane & 15;
  const int rq = (lane >> 4) * 4;
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        ct[(wm * C::WM + i * 16 + rq + r) * C::LDC + wn * C::WN + j * 16 + r16] = acc[i][j][r];
}

// ---------------------------------------------------------------------------
// CONV mode
// ---------------------------------------------------------------------------

template <class C>
__global__ __launch_bounds__(C::NT) void igemm_conv(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[C::LDS_BYTES];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % C::WAVES_M;
  const int wn = wave / C::WAVES_M;

  const int tilesN = (a.N + C::BN - 1) / C::BN;
  const int nb = gridDim.x;
  const int bid = xcd_remap(blockIdx.x, nb);
  const int tn = bid % tilesN;
  const int tm = bid / tilesN;
  const long m0 = (long)tm * C::BM;
  const int n0 = tn * C::BN;

  const int H = a.g.H, W = a.g.W, HW = a.g.H * a.g.W;
  const long P = a.g.pixels();

  // this thread's A rows: pixel index and the 9-bit mask of in-image taps
  const int kv = tid % C::KV;
  long ppix[C::NVA];
  uint32_t pmask[C::NVA];
#pragma unroll
  for (int j = 0; j < C::NVA; ++j) {
    const long m = m0 + tid / C::KV + j * (C::NT / C::KV);
    ppix[j] = m;
    uint32_t mask = 0;
    if (m < P) {
      const int img = (int)(m / HW);
      const int rem = (int)(m - (long)img * HW);
      const int h = rem / W;
      const int w = rem - h * W;
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const int hh = h + t / 3 - 1, ww = w + t % 3 - 1;
        if (hh >= 0 && hh < H && ww >= 0 && ww < W) mask |= 1u << t;
      }
    }
    pmask[j] = mask;
  }

  VecT<C::F32> ra[C::NVA], rb[C::NVB];
  const Seg sg0 = a.seg[0], sg1 = a.seg[1], sg2 = a.seg[2];
  const int nseg = a.nseg;

  auto load_a = [&](const Seg& sg, int k0) __attribute__((always_inline)) {
    const int r = k0 - sg.begin;
    const int tap = r / sg.C;
    const int cb = r - tap * sg.C + kv * 8;
    // the centre tap of a 3x3 segment and every 1x1 tap read the pixel itself
    const int t9 = sg.taps == 9 ? tap : 4;
    const long shift = (long)(t9 / 3 - 1) * W + (t9 % 3 - 1);
#pragma unroll
    for (int j = 0; j < C::NVA; ++j) {
      if ((pmask[j] >> t9) & 1u)
        vload<C::F32>(vaddr<C::F32>(sg.in, ppix[j] + shift, cb), ra[j]);
      else
        vzero<C::F32>(ra[j]);
    }
  };

  auto load_tiles = [&](int kt) __attribute__((always_inline)) {
    const int k0 = kt * C::BK;
    // the segment is uniform across the block; branch so every access to the
    // segment table uses a constant index
    const int s = seg_of(nseg, sg1.begin, sg2.begin, k0);
    if (s == 0)
      load_a(sg0, k0);
    else if (s == 1)
      load_a(sg1, k0);
    else
      load_a(sg2, k0);
#pragma unroll
    for (int j = 0; j < C::NVB; ++j) {
      const int n = n0 + tid / C::KV + j * (C::NT / C::KV);
      if (n < a.N)
        vload<C::F32>(static_cast<const char*>(a.Bw) + ((long)n * a.ldb + k0 + kv * 8) * C::ESZ,
                      rb[j]);
      else
        vzero<C::F32>(rb[j]);
    }
  };

  auto store_tiles = [&](int buf) __attribute__((always_inline)) {
    char* As = smem + buf * (C::LDS_A + C::LDS_B);
    char* Bs = As + C::LDS_A;
#pragma unroll
    for (int j = 0; j < C::NVA; ++j)
      lds_put<C>(As, tid / C::KV + j * (C::NT / C::KV), kv * 8, ra[j]);
#pragma unroll
    for (int j = 0; j < C::NVB; ++j)
      lds_put<C>(Bs, tid / C::KV + j * (C::NT / C::KV), kv * 8, rb[j]);
  };

  f32x4_t acc[C::TM][C::TN];
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int KT = a.K / C::BK;
  load_tiles(0);
  store_tiles(0);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    if (kt + 1 < KT) load_tiles(kt + 1);
    const char* As = smem + (kt & 1) * (C::LDS_A + C::LDS_B);
    mma_tile<C>(As, As + C::LDS_A, wm, wn, lane, acc);
    if (kt + 1 < KT) store_tiles((kt + 1) & 1);
    __syncthreads();
  }

  // epilogue: accumulators -> LDS -> rows of 8 channels (+bias, +rowvec,
  // +residual) -> 16-byte stores
  float* ct = reinterpret_cast<float*>(smem);
  acc_to_lds<C>(ct, wm, wn, lane, acc);
  __syncthreads();
  constexpr int NV8 = C::BN / 8;
  for (int i = tid; i < C::BM * NV8; i += C::NT) {
    const int row = i / NV8;
    const int n = n0 + (i - row * NV8) * 8;
    const long m = m0 + row;
    if (m >= P || n >= a.N) continue;
    const float* src = ct + row * C::LDC + (n - n0);
    float v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = src[q];
    if (a.bias) {
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] += a.bias[n + q];
    }
    if (a.rowvec) {
      const float* rv = a.rowvec + (long)(m / HW) * a.N + n;
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] += rv[q];
    }
    if (a.resid.s0.ptr) {
      float r[8];
      ld8(a.resid.s0, m, n, r);
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] += r[q];
    }
    st8(a.out, a.out_dtype, a.ldo, m, n, v);
    if (a.out2) st8(a.out2, a.out_dtype, a.ldo, m, n, v);
  }
}

// ---------------------------------------------------------------------------
// WGRAD mode
// ---------------------------------------------------------------------------

template <class C>
__global__ __launch_bounds__(C::NT) void igemm_wgrad(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[C::LDS_BYTES];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % C::WAVES_M;
  const int wn = wave / C::WAVES_M;

  const int tilesN = (a.N + C::BN - 1) / C::BN;
  const int tn = blockIdx.x % tilesN;
  const int tm = blockIdx.x / tilesN;
  const int m0 = tm * C::BM;
  const int n0 = tn * C::BN;
  const int z = blockIdx.z;

  const int H = a.g.H, W = a.g.W, HW = a.g.H * a.g.W;
  const long P = a.g.pixels();
  const long pbeg = (long)z * a.kchunk;
  const long pend = (pbeg + a.kchunk < P) ? pbeg + a.kchunk : P;
  const Seg sg0 = a.seg[0], sg1 = a.seg[1], sg2 = a.seg[2];
  const int nseg = a.nseg;
  const VIn gy = a.gy;

  VecT<C::F32> rt[C::NMT][8];

  // B micro-tile: 8 columns (one segment, one tap, 8 channels) x 8 pixels
  auto load_b = [&](const Seg& sg, int n, long p, VecT<C::F32> (&in)[8])
      __attribute__((always_inline)) {
    const int r = n - sg.begin;
    const int tap = r / sg.C;
    const int c = r - tap * sg.C;
    const int t9 = sg.taps == 9 ? tap : 4;
    const int oy = t9 / 3 - 1, ox = t9 % 3 - 1;
    int img = (int)(p / HW);
    int rem = (int)(p - (long)img * HW);
    int h = rem / W;
    int w = rem - h * W;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int hh = h + oy, ww = w + ox;
      if (p + e < pend && hh >= 0 && hh < H && ww >= 0 && ww < W)
        vload<C::F32>(vaddr<C::F32>(sg.in, p + e + (long)oy * W + ox, c), in[e]);
      else
        vzero<C::F32>(in[e]);
      if (++w == W) {
        w = 0;
        if (++h == H) {
          h = 0;
          ++img;
        }
      }
    }
  };

  // micro-tile t: t < NMA -> A rows (output channels), else B rows (columns)
  auto load_tiles = [&](long p0) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < C::NMT; ++u) {
      const int t = tid + u * C::NT;
      if (t >= C::NMA + C::NMB) break;
      VecT<C::F32> in[8];
      if (t < C::NMA) {
        const int oi = t / (C::BK / 8), pk = t % (C::BK / 8);
        const int o = m0 + oi * 8;
        const long p = p0 + pk * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          if (o < a.M && p + e < pend)
            vload<C::F32>(vaddr<C::F32>(gy, p + e, o), in[e]);
          else
            vzero<C::F32>(in[e]);
        }
      } else {
        const int tb = t - C::NMA;
        const int ni = tb / (C::BK / 8), pk = tb % (C::BK / 8);
        const int n = n0 + ni * 8;
        const long p = p0 + pk * 8;
        if (n < a.N) {
          const int s = seg_of(nseg, sg1.begin, sg2.begin, n);
          if (s == 0)
            load_b(sg0, n, p, in);
          else if (s == 1)
            load_b(sg1, n, p, in);
          else
            load_b(sg2, n, p, in);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) vzero<C::F32>(in[e]);
        }
      }
      transpose8<C::F32>(in, rt[u]);
    }
  };

  auto store_tiles = [&](int buf) __attribute__((always_inline)) {
    char* As = smem + buf * (C::LDS_A + C::LDS_B);
    char* Bs = As + C::LDS_A;
#pragma unroll
    for (int u = 0; u < C::NMT; ++u) {
      const int t = tid + u * C::NT;
      if (t >= C::NMA + C::NMB) break;
      if (t < C::NMA) {
        const int oi = t / (C::BK / 8), pk = t % (C::BK / 8);
#pragma unroll
        for (int q = 0; q < 8; ++q) lds_put<C>(As, oi * 8 + q, pk * 8, rt[u][q]);
      } else {
        const int tb = t - C::NMA;
        const int ni = tb / (C::BK / 8), pk = tb % (C::BK / 8);
#pragma unroll
        for (int q = 0; q < 8; ++q) lds_put<C>(Bs, ni * 8 + q, pk * 8, rt[u][q]);
      }
    }
  };

  f32x4_t acc[C::TM][C::TN];
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int KT = (int)((pend - pbeg + C::BK - 1) / C::BK);
  if (KT > 0) {
    load_tiles(pbeg);
    store_tiles(0);
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
      if (kt + 1 < KT) load_tiles(pbeg + (long)(kt + 1) * C::BK);
      const char* As = smem + (kt & 1) * (C::LDS_A + C::LDS_B);
      mma_tile<C>(As, As + C::LDS_A, wm, wn, lane, acc);
      if (kt + 1 < KT) store_tiles((kt + 1) & 1);
      __syncthreads();
    }
  }

  // partials through LDS so each row is written as whole 16-byte vectors
  float* ct = reinterpret_cast<float*>(smem);
  acc_to_lds<C>(ct, wm, wn, lane, acc);
  __syncthreads();
  float* part = a.part + (long)z * a.M * a.N;
  constexpr int NV4 = C::BN / 4;
  for (int i = tid; i < C::BM * NV4; i += C::NT) {
    const int row = i / NV4;
    const int n = n0 + (i - row * NV4) * 4;
    const int m = m0 + row;
    if (m >= a.M || n >= a.N) continue;
    const float* src = ct + row * C::LDC + (n - n0);
    *reinterpret_cast<float4*>(part + (long)m * a.N + n) =
        make_float4(src[0], src[1], src[2], src[3]);
  }
}

// Sum the split partials in split order and accumulate into the gradients
// of each segment (rows of length end - begin: OHWI for 3x3, [O][I] for 1x1).
__global__ void wgrad_finalize(GemmArgs a, int splits) {
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)a.M * a.N) return;
  const int m = (int)(idx / a.N);
  const int n = (int)(idx - (long)m * a.N);
  float s = 0.f;
  for (int z = 0; z < splits; ++z) s += a.part[(long)z * a.M * a.N + idx];
  const Seg sg0 = a.seg[0], sg1 = a.seg[1], sg2 = a.seg[2];
  const int si = seg_of(a.nseg, sg1.begin, sg2.begin, n);
  const Seg& sg = si == 0 ? sg0 : (si == 1 ? sg1 : sg2);
  const int len = sg.end - sg.begin;
  sg.grad[(long)m * len + (n - sg.begin)] += s;
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

using CfgBf16 = Cfg<128, 128, 64, 64, 64, false>;
using CfgBf16K32 = Cfg<128, 128, 32, 64, 64, false>;
using CfgF32 = Cfg<64, 64, 32, 32, 32, true>;

template <class C>
static hipError_t launch_conv_t(const GemmArgs& a, hipStream_t st) {
  const long tilesM = (a.g.pixels() + C::BM - 1) / C::BM;
  const long tilesN = (a.N + C::BN - 1) / C::BN;
  hipLaunchKernelGGL(igemm_conv<C>, dim3((unsigned)(tilesM * tilesN)), dim3(C::NT), 0, st, a);
  return hipGetLastError();
}

template <class C>
static hipError_t launch_wgrad_t(GemmArgs a, int splits, hipStream_t st) {
  const long tilesM = (a.M + C::BM - 1) / C::BM;
  const long tilesN = (a.N + C::BN - 1) / C::BN;
  hipLaunchKernelGGL(igemm_wgrad<C>, dim3((unsigned)(tilesM * tilesN), 1, splits),
                     dim3(C::NT), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const long total = (long)a.M * a.N;
  hipLaunchKernelGGL(wgrad_finalize, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st,
                     a, splits);
  return hipGetLastError();
}

// Tile configuration: 0 = bf16 BK 64, 1 = bf16 BK 32, 2 = fp32.
int gemm_bk(int cfg) { return cfg == 2 ? CfgF32::BK : (cfg == 1 ? CfgBf16K32::BK : CfgBf16::BK); }
int gemm_bm(int cfg) { return cfg == 2 ? CfgF32::BM : CfgBf16::BM; }
int gemm_bn(int cfg) { return cfg == 2 ? CfgF32::BN : CfgBf16::BN; }

hipError_t launch_conv(const GemmArgs& a, int cfg, hipStream_t st) {
  switch (cfg) {
    case 0: return launch_conv_t<CfgBf16>(a, st);
    case 1: return launch_conv_t<CfgBf16K32>(a, st);
    default: return launch_conv_t<CfgF32>(a, st);
  }
}

hipError_t launch_wgrad(const GemmArgs& a, int cfg, int splits, hipStream_t st) {
  switch (cfg) {
    case 0: return launch_wgrad_t<CfgBf16>(a, splits, st);
    case 1: return launch_wgrad_t<CfgBf16K32>(a, splits, st);
    default: return launch_wgrad_t<CfgF32>(a, splits, st);
  }
}

}  // namespace pulse
