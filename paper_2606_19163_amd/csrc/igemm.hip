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
  static constexpr int LDS_A = BM * LDK * ESZ;
  static constexpr int LDS_B = BN * LDK * ESZ;
  static constexpr int LDS_OPS = 2 * (LDS_A + LDS_B);
  static constexpr int LDC = BN + 4;              // fp32 epilogue rows
  static constexpr int LDS_EPI = WM * LDC * 4;    // one wave row at a time
  static constexpr int LDS_BYTES = LDS_OPS > LDS_EPI ? LDS_OPS : LDS_EPI;
  // CONV mode: 8-element vectors per thread for the A and B tiles
  static constexpr int NVA = (BM * KV + NT - 1) / NT;
  static constexpr int NVB = (BN * KV + NT - 1) / NT;
  // WGRAD mode: 8x8 micro-tiles per thread
  static constexpr int NMA = (BM / 8) * (BK / 8);
  static constexpr int NMB = (BN / 8) * (BK / 8);
  static constexpr int NMT = (NMA + NMB + NT - 1) / NT;
  static_assert(BM % WM == 0 && BN % WN == 0 && WM % 16 == 0 && WN % 16 == 0, "tile");
  static_assert(BK % 32 == 0 && NT % KV == 0, "BK");
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

// Buffer resource over `bytes` bytes at p: loads at offsets past the end
// return zero, which gives the zero padding without branches.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, long bytes) {
  const int n = bytes > 0x7fffffffL ? 0x7fffffff : (int)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, p ? n : 0,
                                           0x00020000);
}

constexpr uint32_t OOB = 0x80000000u;  // an offset past every buffer

template <bool F32>
__device__ __forceinline__ void bload(__amdgpu_buffer_rsrc_t r, uint32_t off, VecT<F32>& v) {
  const auto q0 = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
  v.w[0] = q0.x; v.w[1] = q0.y; v.w[2] = q0.z; v.w[3] = q0.w;
  if constexpr (F32) {
    const auto q1 =
        __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off + 16u, 0, 0));
    v.w[F32 ? 4 : 0] = q1.x; v.w[F32 ? 5 : 1] = q1.y;
    v.w[F32 ? 6 : 2] = q1.z; v.w[F32 ? 7 : 3] = q1.w;
  }
}

// Per-segment constants of a kernel launch, kept in scalar registers: the
// buffer resources of its one or two sources, their pixel pitch in bytes and
// the channel split.
struct SegRt {
  __amdgpu_buffer_rsrc_t r0, r1;
  uint32_t pitch0, pitch1;
  int c0, C, taps, begin;
};

template <bool F32>
__device__ __forceinline__ SegRt seg_rt(const Seg& g, long P) {
  constexpr int esz = F32 ? 4 : 2;
  SegRt s;
  s.r0 = make_rsrc(g.in.s0.ptr, P * g.in.s0.C * esz);
  s.r1 = make_rsrc(g.in.s1.ptr, P * g.in.s1.C * esz);
  s.pitch0 = (uint32_t)(g.in.s0.C * esz);
  s.pitch1 = (uint32_t)(g.in.s1.C * esz);
  s.c0 = g.in.c0;
  s.C = g.C;
  s.taps = g.taps;
  s.begin = g.begin;
  return s;
}

__device__ __forceinline__ SegRt pick(int s, const SegRt& a, const SegRt& b, const SegRt& c) {
  return s == 0 ? a : (s == 1 ? b : c);
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
// Workgroups are dispatched round-robin over the 8 XCDs (block b on XCD
// b % 8).  Map them so that XCD x runs one contiguous range of logical
// blocks: XCD x holds q + (x < r) blocks for nb = 8 q + r.
__device__ __forceinline__ int xcd_remap(int bid, int nb) {
  const int q = nb >> 3, r = nb & 7, x = bid & 7;
  return x * q + (x < r ? x : r) + (bid >> 3);
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

// Park one wave's accumulators in an fp32 [WM][LDC] LDS tile (rows of the
// wave's row group, columns of the whole block tile).
template <class C>
__device__ __forceinline__ void acc_to_lds(float* ct, int wn, int lane,
                                           const f32x4_t (&acc)[C::TM][C::TN]) {
  const int r16 = lane & 15;
  const int rq = (lane >> 4) * 4;
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        ct[(i * 16 + rq + r) * C::LDC + wn * C::WN + j * 16 + r16] = acc[i][j][r];
}

// ---------------------------------------------------------------------------
// CONV mode
// ---------------------------------------------------------------------------

template <class C>
__global__ __launch_bounds__(C::NT) void igemm_conv(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[C::LDS_BYTES];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar registers
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
  // (rows past the tile or past P get an empty mask and read zeros)
  const int kv = tid % C::KV;
  uint32_t ppix[C::NVA];
  uint32_t pmask[C::NVA];
#pragma unroll
  for (int j = 0; j < C::NVA; ++j) {
    const int rowt = tid / C::KV + j * (C::NT / C::KV);
    const long m = rowt < C::BM ? m0 + rowt : P;
    ppix[j] = (uint32_t)m;
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
  // weight rows of this thread (rows past N read as zeros)
  uint32_t boff[C::NVB];
#pragma unroll
  for (int j = 0; j < C::NVB; ++j) {
    const int rowt = tid / C::KV + j * (C::NT / C::KV);
    const int n = n0 + rowt;
    boff[j] = (rowt < C::BN && n < a.N) ? (uint32_t)((long)n * a.ldb * C::ESZ + kv * 8 * C::ESZ)
                                        : OOB;
  }

  VecT<C::F32> ra[C::NVA], rb[C::NVB];
  const int nseg = a.nseg;
  const SegRt q0 = seg_rt<C::F32>(a.seg[0], P);
  const SegRt q1 = seg_rt<C::F32>(a.seg[1], P);
  const SegRt q2 = seg_rt<C::F32>(a.seg[2], P);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.Bw, (long)a.N * a.ldb * C::ESZ);

  auto load_tiles = [&](int kt) __attribute__((always_inline)) {
    const int k0 = kt * C::BK;
    // everything below up to the loads is uniform across the block
    const SegRt q = pick(seg_of(nseg, q1.begin, q2.begin, k0), q0, q1, q2);
    const int r = k0 - q.begin;
    const int tap = r / q.C;
    const int cb = r - tap * q.C;
    const bool second = cb >= q.c0;
    const __amdgpu_buffer_rsrc_t rs = second ? q.r1 : q.r0;
    const uint32_t pitch = second ? q.pitch1 : q.pitch0;
    const uint32_t coff = (uint32_t)(((second ? cb - q.c0 : cb) + kv * 8) * C::ESZ);
    // the centre tap of a 3x3 segment and every 1x1 tap read the pixel itself
    const int t9 = q.taps == 9 ? tap : 4;
    const int shift = (t9 / 3 - 1) * W + (t9 % 3 - 1);
#pragma unroll
    for (int j = 0; j < C::NVA; ++j) {
      const uint32_t off = ((pmask[j] >> t9) & 1u) ? (ppix[j] + shift) * pitch + coff : OOB;
      bload<C::F32>(rs, off, ra[j]);
    }
    const uint32_t kb = (uint32_t)(k0 * C::ESZ);
#pragma unroll
    for (int j = 0; j < C::NVB; ++j) bload<C::F32>(rw, boff[j] + kb, rb[j]);
  };

  auto store_tiles = [&](int buf) __attribute__((always_inline)) {
    char* As = smem + buf * (C::LDS_A + C::LDS_B);
    char* Bs = As + C::LDS_A;
#pragma unroll
    for (int j = 0; j < C::NVA; ++j) {
      const int rowt = tid / C::KV + j * (C::NT / C::KV);
      if ((C::BM * C::KV) % C::NT == 0 || rowt < C::BM) lds_put<C>(As, rowt, kv * 8, ra[j]);
    }
#pragma unroll
    for (int j = 0; j < C::NVB; ++j) {
      const int rowt = tid / C::KV + j * (C::NT / C::KV);
      if ((C::BN * C::KV) % C::NT == 0 || rowt < C::BN) lds_put<C>(Bs, rowt, kv * 8, rb[j]);
    }
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

  // epilogue, one wave row group at a time: accumulators -> LDS -> rows of
  // 8 channels (+bias, +rowvec, +residual) -> 16-byte stores
  float* ct = reinterpret_cast<float*>(smem);
  constexpr int NV8 = C::BN / 8;
#pragma unroll 1
  for (int g = 0; g < C::WAVES_M; ++g) {
    if (wm == g) acc_to_lds<C>(ct, wn, lane, acc);
    __syncthreads();
    for (int i = tid; i < C::WM * NV8; i += C::NT) {
      const int row = i / NV8;
      const int n = n0 + (i - row * NV8) * 8;
      const long m = m0 + g * C::WM + row;
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
    __syncthreads();
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
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar registers
  const int wm = wave % C::WAVES_M;
  const int wn = wave / C::WAVES_M;

  // Block -> (split, tile), split-major over a contiguous range per XCD,
  // so the blocks of one pixel split share that XCD's L2.
  const int tilesN = (a.N + C::BN - 1) / C::BN;
  const int ntiles = ((a.M + C::BM - 1) / C::BM) * tilesN;
  const int lb = xcd_remap(blockIdx.x, gridDim.x);
  const int z = lb / ntiles;
  const int tile = lb - z * ntiles;
  const int tn = tile % tilesN;
  const int tm = tile / tilesN;
  const int m0 = tm * C::BM;
  const int n0 = tn * C::BN;

  const int H = a.g.H, W = a.g.W, HW = a.g.H * a.g.W;
  const long P = a.g.pixels();
  const long pbeg = (long)z * a.kchunk;
  const long pend = (pbeg + a.kchunk < P) ? pbeg + a.kchunk : P;
  const int nseg = a.nseg;
  const SegRt q0 = seg_rt<C::F32>(a.seg[0], P);
  const SegRt q1 = seg_rt<C::F32>(a.seg[1], P);
  const SegRt q2 = seg_rt<C::F32>(a.seg[2], P);
  const __amdgpu_buffer_rsrc_t rg = make_rsrc(a.gy.s0.ptr, P * a.gy.s0.C * C::ESZ);
  const uint32_t gpitch = (uint32_t)(a.gy.s0.C * C::ESZ);

  // this thread's micro-tiles, loaded raw (pixel-major) and transposed when
  // they are written to LDS
  VecT<C::F32> rt[C::NMT][8];

  // B micro-tile: 8 columns (one segment, one tap, 8 channels) x 8 pixels
  auto load_b = [&](int n, long p, VecT<C::F32> (&in)[8]) __attribute__((always_inline)) {
    const SegRt q = pick(seg_of(nseg, q1.begin, q2.begin, n), q0, q1, q2);
    const int r = n - q.begin;
    const int tap = r / q.C;
    const int c = r - tap * q.C;
    const bool second = c >= q.c0;
    const __amdgpu_buffer_rsrc_t rs = second ? q.r1 : q.r0;
    const uint32_t pitch = second ? q.pitch1 : q.pitch0;
    const uint32_t coff = (uint32_t)((second ? c - q.c0 : c) * C::ESZ);
    const int t9 = q.taps == 9 ? tap : 4;
    const int oy = t9 / 3 - 1, ox = t9 % 3 - 1;
    const int img = (int)(p / HW);
    const int rem = (int)(p - (long)img * HW);
    const int h = rem / W;
    const int w = rem - h * W;
    if (W % 8 == 0) {
      // the 8 pixels share one image row
      const bool rowok = h + oy >= 0 && h + oy < H;
      const uint32_t base = (uint32_t)(p + oy * W + ox);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const bool ok = rowok && p + e < pend && w + e + ox >= 0 && w + e + ox < W;
        bload<C::F32>(rs, ok ? (base + e) * pitch + coff : OOB, in[e]);
      }
    } else {
      int hh = h, ww = w;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const bool ok = p + e < pend && hh + oy >= 0 && hh + oy < H && ww + ox >= 0 &&
                        ww + ox < W;
        bload<C::F32>(rs, ok ? (uint32_t)(p + e + oy * W + ox) * pitch + coff : OOB, in[e]);
        if (++ww == W) {
          ww = 0;
          if (++hh == H) hh = 0;
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
      if (t < C::NMA) {
        const int oi = t / (C::BK / 8), pk = t % (C::BK / 8);
        const int o = m0 + oi * 8;
        const long p = p0 + pk * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const bool ok = o < a.M && p + e < pend;
          bload<C::F32>(rg, ok ? (uint32_t)(p + e) * gpitch + o * C::ESZ : OOB, rt[u][e]);
        }
      } else {
        const int tb = t - C::NMA;
        const int ni = tb / (C::BK / 8), pk = tb % (C::BK / 8);
        const int n = n0 + ni * 8;
        const long p = p0 + pk * 8;
        if (n < a.N) {
          load_b(n, p, rt[u]);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) vzero<C::F32>(rt[u][e]);
        }
      }
    }
  };

  auto store_tiles = [&](int buf) __attribute__((always_inline)) {
    char* As = smem + buf * (C::LDS_A + C::LDS_B);
    char* Bs = As + C::LDS_A;
#pragma unroll
    for (int u = 0; u < C::NMT; ++u) {
      const int t = tid + u * C::NT;
      if (t >= C::NMA + C::NMB) break;
      VecT<C::F32> tr[8];
      transpose8<C::F32>(rt[u], tr);
      if (t < C::NMA) {
        const int oi = t / (C::BK / 8), pk = t % (C::BK / 8);
#pragma unroll
        for (int q = 0; q < 8; ++q) lds_put<C>(As, oi * 8 + q, pk * 8, tr[q]);
      } else {
        const int tb = t - C::NMA;
        const int ni = tb / (C::BK / 8), pk = tb % (C::BK / 8);
#pragma unroll
        for (int q = 0; q < 8; ++q) lds_put<C>(Bs, ni * 8 + q, pk * 8, tr[q]);
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

  // partials through LDS (one wave row group at a time) so each row is
  // written as whole 16-byte vectors
  float* ct = reinterpret_cast<float*>(smem);
  float* part = a.part + (long)z * a.M * a.N;
  constexpr int NV4 = C::BN / 4;
#pragma unroll 1
  for (int g = 0; g < C::WAVES_M; ++g) {
    if (wm == g) acc_to_lds<C>(ct, wn, lane, acc);
    __syncthreads();
    for (int i = tid; i < C::WM * NV4; i += C::NT) {
      const int row = i / NV4;
      const int n = n0 + (i - row * NV4) * 4;
      const int m = m0 + g * C::WM + row;
      if (m >= a.M || n >= a.N) continue;
      const float* src = ct + row * C::LDC + (n - n0);
      *reinterpret_cast<float4*>(part + (long)m * a.N + n) =
          make_float4(src[0], src[1], src[2], src[3]);
    }
    __syncthreads();
  }
}

// Sum the split partials in split order and accumulate into the gradients
// of each segment (rows of length end - begin: OHWI for 3x3, [O][I] for 1x1).
// Four consecutive columns per thread (N and the segment bounds are
// multiples of 8).
__global__ void wgrad_finalize(GemmArgs a, int splits) {
  const long idx = ((long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (idx >= (long)a.M * a.N) return;
  const int m = (int)(idx / a.N);
  const int n = (int)(idx - (long)m * a.N);
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int z = 0; z < splits; ++z) {
    const float4 v = *reinterpret_cast<const float4*>(a.part + (long)z * a.M * a.N + idx);
    s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
  }
  const Seg sg0 = a.seg[0], sg1 = a.seg[1], sg2 = a.seg[2];
  const int si = seg_of(a.nseg, sg1.begin, sg2.begin, n);
  const Seg& sg = si == 0 ? sg0 : (si == 1 ? sg1 : sg2);
  const int len = sg.end - sg.begin;
  float* g = sg.grad + (long)m * len + (n - sg.begin);
  g[0] += s.x; g[1] += s.y; g[2] += s.z; g[3] += s.w;
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

// Tile shapes.  bf16 with 64 channels per K-step unless noted.
using T128x128K32 = Cfg<128, 128, 32, 64, 64, false>; // channel counts % 64 != 0
using T64x64F32 = Cfg<64, 64, 32, 32, 32, true>;      // the fp32 stage

template <class C>
static hipError_t launch_conv_t(const GemmArgs& a, hipStream_t st) {
  const long tilesM = (a.g.pixels() + C::BM - 1) / C::BM;
  const long tilesN = (a.N + C::BN - 1) / C::BN;
  hipLaunchKernelGGL(igemm_conv<C>, dim3((unsigned)(tilesM * tilesN)), dim3(C::NT), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_wgrad_finalize(const GemmArgs& a, int splits, hipStream_t st) {
  const long total = (long)a.M * a.N / 4;
  hipLaunchKernelGGL(wgrad_finalize, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st,
                     a, splits);
  return hipGetLastError();
}

template <class C>
static hipError_t launch_wgrad_t(GemmArgs a, int splits, hipStream_t st) {
  const long tilesM = (a.M + C::BM - 1) / C::BM;
  const long tilesN = (a.N + C::BN - 1) / C::BN;
  hipLaunchKernelGGL(igemm_wgrad<C>, dim3((unsigned)(tilesM * tilesN * splits)), dim3(C::NT), 0,
                     st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const long total = (long)a.M * a.N / 4;
  hipLaunchKernelGGL(wgrad_finalize, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st,
                     a, splits);
  return hipGetLastError();
}

template <class C>
static TileInfo info_t() {
  return TileInfo{C::BM, C::BN, C::BK, 0};
}

TileInfo tile_info(int t) {
  return t == TILE_64x64_F32 ? info_t<T64x64F32>() : info_t<T128x128K32>();
}

hipError_t launch_conv(const GemmArgs& a, int t, hipStream_t st) {
  return t == TILE_64x64_F32 ? launch_conv_t<T64x64F32>(a, st) : launch_conv_t<T128x128K32>(a, st);
}

hipError_t launch_wgrad(const GemmArgs& a, int t, int splits, hipStream_t st) {
  return t == TILE_64x64_F32 ? launch_wgrad_t<T64x64F32>(a, splits, st)
                             : launch_wgrad_t<T128x128K32>(a, splits, st);
}

}  // namespace pulse
