// Implicit-GEMM convolution, second generation: operand tiles move from
// HBM/L2 to LDS with the LDS-DMA loads of gfx950 (buffer_load ... lds /
// global_load_lds_dwordx4), so no register staging and no VALU touch the
// operands on their way to the matrix cores, and two LDS stages overlap the
// next tile's loads with the current tile's MFMAs.
//
// A wave-wide DMA load writes 64 lanes x 16 bytes contiguously (lane i at
// base + 16 i), so every tile is a dense array of 16-byte chunks and bank
// conflicts are avoided by XOR-swizzling the chunk index instead of padding.
//
//  * CONV mode (forward, data gradient): tiles are K-contiguous rows of 64
//    bf16 (128 bytes): A rows are pixels, B rows are output channels.
//    Fragments are read with ds_read_b128.  Out-of-image taps and rows past
//    the tile read as zero through out-of-range buffer offsets.
//  * WGRAD mode: both tiles keep the NHWC order, rows of channels per pixel
//    ([64 pixels][BM] and [64 pixels][BN]); the MFMA wants 8 consecutive
//    pixels per lane, which ds_read_b64_tr_b16 delivers (two per fragment):
//    within 16 lanes, lane j receives element j%4 of the rows addressed by
//    lanes 4q + j/4, q = 0..3.  B columns may mix sources within one tile, so
//    its DMA uses per-lane global addresses; invalid elements point at a
//    zeroed 16-byte word.
#include <hip/hip_ext.h>

#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace pulse {

namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;

constexpr uint32_t OOB = 0x80000000u;  // an offset past every buffer

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, long bytes) {
  const int n = bytes > 0x7fffffffL ? 0x7fffffff : (int)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, p ? n : 0,
                                           0x00020000);
}

__device__ __forceinline__ lds_ptr_t lds(char* p) { return (lds_ptr_t)p; }

// s_waitcnt vmcnt(n) (gfx9 encoding; expcnt and lgkmcnt left at their maxima)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}


}  // namespace

template <int BM_, int BN_, int WM_, int WN_, int STAGES_ = 2, int BK_ = 64>
struct CfgC {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, BK = BK_, STAGES = STAGES_;
  static constexpr int WAVES_M = BM / WM, WAVES_N = BN / WN, NW = WAVES_M * WAVES_N;
  static constexpr int NT = NW * 64;
  static constexpr int TM = WM / 16, TN = WN / 16;
  static constexpr int RB = BK * 2;           // row bytes
  static constexpr int CPR = RB / 16;         // 16-byte chunks per row
  static constexpr int RPL = 1024 / RB;       // rows per 1 KB wave load
  static constexpr int KH = BK / 32;          // MFMA K-steps (32) per stage
  static constexpr int A_BYTES = BM * RB, B_BYTES = BN * RB;
  static constexpr int STAGE = A_BYTES + B_BYTES;
  static constexpr int WLA = A_BYTES / 1024, WLB = B_BYTES / 1024, WL = WLA + WLB;
  static constexpr int NU = (WL + NW - 1) / NW;  // loads of waves < REM (all when REM == 0)
  static constexpr int REM = WL % NW;
  static constexpr int NU_LO = WL / NW;           // loads of waves >= REM
  static constexpr int UA = WLA / NW;  // loads u < UA fill A, the rest fill B
  static constexpr int LDC = BN + 4;
  static constexpr int LDS_BYTES = STAGES * STAGE;
  static_assert(BK == 32 || BK == 64, "K-step");
  static_assert(STAGES >= 2 && STAGES <= 4, "stages");
  static_assert(16 * LDC * 4 <= STAGES * STAGE, "epilogue slice must fit the stages");
  static_assert((2 * 16 * LDC + 4 * BN) * 4 <= STAGES * STAGE,
                "GroupNorm-backward slices and constants must fit the stages");
  static_assert(STAGES * STAGE <= 160 * 1024, "LDS");
  static_assert(A_BYTES % 1024 == 0 && B_BYTES % 1024 == 0, "whole wave loads");
  static_assert(WLA % NW == 0, "A wave loads must split evenly over the waves");
  static_assert(A_BYTES + (TN - 1) * 16 * RB < 65536, "fragment offsets are 16-bit immediates");
  static_assert(KH * (TM + TN) <= 15 || KH == 2, "lgkmcnt");
  static_assert(BM % 16 == 0 && BN % 16 == 0 && WM % 16 == 0 && WN % 16 == 0, "tile");
};

// Row swizzle of conv tiles: chunk c of row r lives in slot c ^ swz(r).  With
// 128-byte rows, rows r and r+1 fall in opposite halves of the 256-byte bank
// period and the swizzle separates rows of equal parity; with 64-byte rows,
// four rows share a period and the swizzle separates rows r and r+4k.
template <int RB>
__device__ __forceinline__ int swz_row(int r) {
  return RB == 128 ? ((r >> 1) & 7) : ((r >> 2) & 3);
}

// Weight-gradient tiles are pixel-major rows of P bytes.  Row r is stored
// rotated by rot(r) = a (r & 3) + b ((r >> 3) & 1) units of 32 bytes (16
// channels), chosen so that each half-wave of a transpose read (rows
// {0..3, 8..11} or {16..19, 24..27} of a 32-row slice, 32 bytes per row) hits
// 8 distinct 32-byte bank groups of the 64-bank LDS.
constexpr int rot_conflicts(int P, int a, int b) {
  const int U = P / 32;
  int bad = 0;
  for (int s = 0; s < 2; ++s)
    for (int h = 0; h < 2; ++h)
      for (int hw = 0; hw < 2; ++hw)
        for (int u = 0; u < U; ++u) {
          int seen = 0;
          for (int g = 2 * hw; g < 2 * hw + 2; ++g)
            for (int q = 0; q < 4; ++q) {
              const int r = 32 * s + 4 * h + 8 * g + q;
              const int grp = (r * U + (u + a * (r & 3) + b * ((r >> 3) & 1)) % U) % 8;
              if ((seen >> grp) & 1) ++bad;
              seen |= 1 << grp;
            }
        }
  return bad;
}
constexpr int best_rot(int P) {  // a + 256 * b of the first conflict-free pair
  const int U = P / 32;
  int best = 0, best_bad = 1 << 30;
  for (int a = 0; a < U; ++a)
    for (int b = 0; b < U; ++b) {
      const int bad = rot_conflicts(P, a, b);
      if (bad < best_bad) {
        best_bad = bad;
        best = a + 256 * b;
      }
      if (bad == 0) return best;
    }
  return best;
}

template <int BM_, int BN_, int WM_, int WN_>
struct CfgW {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, BK = 64;
  static constexpr int WAVES_M = BM / WM, WAVES_N = BN / WN, NW = WAVES_M * WAVES_N;
  static constexpr int NT = NW * 64;
  static constexpr int TM = WM / 16, TN = WN / 16;
  static constexpr int PA = BM * 2, PB = BN * 2;  // row pitch (bytes): one pixel
  static constexpr int CA = BM / 8, CB = BN / 8;  // 16-byte chunks per row
  static constexpr int A_BYTES = BK * PA, B_BYTES = BK * PB;
  static constexpr int STAGE = A_BYTES + B_BYTES;
  static constexpr int WLA = A_BYTES / 1024, WLB = B_BYTES / 1024, WL = WLA + WLB;
  static constexpr int NU = WL / NW;
  static constexpr int UA = WLA / NW;  // loads u < UA fill A, the rest fill B
  static constexpr int RA = best_rot(PA), RB = best_rot(PB);
  static constexpr int RA_A = RA % 256, RA_B = RA / 256, RB_A = RB % 256, RB_B = RB / 256;
  static constexpr int LDC = BN + 4;
  static constexpr int LDS_BYTES = 2 * STAGE;
  static_assert(16 * LDC * 4 <= STAGE, "epilogue slice must fit one stage");
  static_assert(2 * STAGE <= 160 * 1024, "LDS");
  static_assert(WL % NW == 0 && WLA % NW == 0 && (BK * PA) % 1024 == 0 &&
                    (BK * PB) % 1024 == 0,
                "loads");
  static_assert(BM % 16 == 0 && BN % 16 == 0, "rows of whole 32-byte units");
  static_assert(36 * PA < 65536 && A_BYTES + 36 * PB < 65536, "read offsets are immediates");
  static_assert(WM % 16 == 0 && WN % 16 == 0, "tile");
};

namespace {

__device__ __forceinline__ int seg_of(int nseg, int b1, int b2, int i) {
  int s = 0;
  if (nseg > 1 && i >= b1) s = 1;
  if (nseg > 2 && i >= b2) s = 2;
  return s;
}

// Workgroups are dispatched round-robin over the 8 XCDs (block b on XCD
// b % 8).  Map them so that XCD x runs one contiguous range of logical
// blocks: XCD x holds q + (x < r) blocks for nb = 8 q + r.
__device__ __forceinline__ int xcd_remap(int bid, int nb) {
  const int q = nb >> 3, r = nb & 7, x = bid & 7;
  return x * q + (x < r ? x : r) + (bid >> 3);
}

// n / d with the launcher's reciprocal M of d (rcp_u32): a multiply-high,
// or a divide where M is 0
__device__ __forceinline__ uint32_t div_rcp(uint32_t n, uint32_t d, uint32_t M) {
  return M ? __umulhi(n, M) : (d < 2 ? n : n / d);
}

__device__ __forceinline__ uint32_t lds_u32(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}

// ds_read_b128 at addr + OFF.  Issued as inline asm so that the compiler's
// waitcnt pass, which cannot tell LDS-DMA targets apart, does not insert a
// vmcnt(0) before it: the kernel waits for its own DMA stages and for these
// reads explicitly (lgkm_wait + tie).
template <int OFF>
__device__ __forceinline__ bf16x8_t ds_rd128(uint32_t addr) {
  bf16x8_t v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF));
  return v;
}

template <int N, int STRIDE, int BASE>
__device__ __forceinline__ void ds_rd_n(bf16x8_t* dst, uint32_t addr) {
  if constexpr (N > 0) {
    ds_rd_n<N - 1, STRIDE, BASE>(dst, addr);
    dst[N - 1] = ds_rd128<BASE + (N - 1) * STRIDE>(addr);
  }
}

// s_waitcnt lgkmcnt(n) (vmcnt and expcnt left at their maxima)
template <int N>
__device__ __forceinline__ void lgkm_wait() {
  static_assert(N >= 0 && N < 16, "lgkmcnt");
  __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (N << 8) | (3 << 14));
}

// Order a value after the preceding waits: the MFMAs that consume it cannot
// be scheduled above them.
__device__ __forceinline__ void tie(bf16x8_t& v) { asm volatile("" : "+v"(v)); }
__device__ __forceinline__ void tie(v4s& v) { asm volatile("" : "+v"(v)); }

// ds_read_b64_tr_b16 at addr + OFF (see ds_rd128 for why it is inline asm)
template <int OFF>
__device__ __forceinline__ v4s ds_rdtr(uint32_t addr) {
  v4s v;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF));
  return v;
}

// 16-byte chunk slot of logical chunk lc in row r of a rotated tile (C
// chunks per row, rotation a (r & 3) + b ((r >> 3) & 1) units of 2 chunks)
__device__ __forceinline__ int rot_slot(int lc, int r, int C, int a, int b) {
  int p = lc + 2 * (a * (r & 3) + b * ((r >> 3) & 1));
  while (p >= C) p -= C;
  return p;
}
__device__ __forceinline__ int rot_logical(int pc, int r, int C, int a, int b) {
  int p = pc - 2 * (a * (r & 3) + b * ((r >> 3) & 1));
  while (p < 0) p += C;
  return p;
}

struct SegRt {
  __amdgpu_buffer_rsrc_t r0, r1;
  uint32_t pitch0, pitch1;
  int c0, C, taps, begin;
};

__device__ __forceinline__ SegRt seg_rt(const Seg& g, long P) {
  SegRt s;
  s.r0 = make_rsrc(g.in.s0.ptr, P * g.in.s0.C * 2);
  s.r1 = make_rsrc(g.in.s1.ptr, P * g.in.s1.C * 2);
  s.pitch0 = (uint32_t)(g.in.s0.C * 2);
  s.pitch1 = (uint32_t)(g.in.s1.C * 2);
  s.c0 = g.in.c0;
  s.C = g.C;
  s.taps = g.taps;
  s.begin = g.begin;
  return s;
}

// field-wise select (a select of whole structs can end up in scratch memory)
__device__ __forceinline__ void select_into(SegRt& d, bool c, const SegRt& a, const SegRt& b) {
  d.r0 = c ? a.r0 : b.r0;
  d.r1 = c ? a.r1 : b.r1;
  d.pitch0 = c ? a.pitch0 : b.pitch0;
  d.pitch1 = c ? a.pitch1 : b.pitch1;
  d.c0 = c ? a.c0 : b.c0;
  d.C = c ? a.C : b.C;
  d.taps = c ? a.taps : b.taps;
  d.begin = c ? a.begin : b.begin;
}

// Stage the accumulator rows [i*16, i*16+16) of every wave of row group g
// into an fp32 [16][LDC] LDS tile.
template <int TM, int TN, int WN, int LDC>
__device__ __forceinline__ void acc16_to_lds(float* ct, int wn, int lane, int i,
                                             const f32x4_t (&acc)[TM][TN]) {
  const int r16 = lane & 15;
  const int rq = (lane >> 4) * 4;
#pragma unroll
  for (int ii = 0; ii < TM; ++ii) {
    if (ii != i) continue;
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) ct[(rq + r) * LDC + wn * WN + j * 16 + r16] = acc[ii][j][r];
  }
}

}  // namespace

// ---------------------------------------------------------------------------
// CONV mode
// ---------------------------------------------------------------------------

// GNB: the instance that writes the GroupNorm-backward sums (a.gnb) of a
// plain output (no bias, timestep row, residual, copy, statistics or K
// split); the others never do, so neither pays for the other's registers.
template <class C, bool GNB = false>
__global__ __launch_bounds__(C::NT) void igemm2_conv(GemmArgs a) {
  // the body exists for the device pass only (the host pass emits the launch stub)
#if defined(__HIP_DEVICE_COMPILE__)
  __shared__ __attribute__((aligned(1024))) char smem[C::STAGES * C::STAGE];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar registers
  const int wm = wave % C::WAVES_M;
  const int wn = wave / C::WAVES_M;

  // block -> (K split, tile), split-major over a contiguous range per XCD
  const int H = a.g.H, W = a.g.W, HW = a.g.H * a.g.W;
  const long P = a.g.pixels();
  const int tilesN = (a.N + C::BN - 1) / C::BN;
  const int ntiles = (int)((P + C::BM - 1) / C::BM) * tilesN;
  const int lb = xcd_remap(blockIdx.x, gridDim.x);
  const int z = (int)div_rcp((uint32_t)lb, (uint32_t)ntiles, a.rcp_nt);
  const int bid = lb - z * ntiles;
  // Tile order within the XCD's range.  Up to 8 column tiles: row-major, a
  // row tile's A rows are reused across all of N and B is small.  Wider N:
  // groups of 8 row tiles swept column by column, so that the blocks an XCD
  // runs together share both their A rows and their B columns in its L2
  // (row-major would stream the whole B through L2 once per row tile).
  int tn, tm;
  if (tilesN <= 8) {
    tm = (int)div_rcp((uint32_t)bid, (uint32_t)tilesN, a.rcp_tn);
    tn = bid - tm * tilesN;
  } else {
    constexpr int GM = 8;
    const int tilesM = ntiles / tilesN;
    const int grp = bid / (GM * tilesN);
    const int first = grp * GM;
    const int gm = min(GM, tilesM - first);
    const int local = bid - grp * GM * tilesN;
    tm = first + local % gm;
    tn = local / gm;
  }
  const long m0 = (long)tm * C::BM;
  const int n0 = tn * C::BN;
  const int KT_ALL = a.K / C::BK;
  const int kt0 = z * a.ksteps;
  const int KT = min(KT_ALL, kt0 + a.ksteps) - kt0;  // K-steps of this block

  // this lane's wave loads: wl = wave + u * NW; A rows first, then B rows.
  // Lane (row rl = lane / 8 of the load, slot lane % 8) fetches logical chunk
  // (lane % 8) ^ swz(row).
  // Image row and column of a tile pixel without divides: the tile's first
  // pixel is at offset rem0 of its image, pixel m0 + r at rem0 + r < HW + BM,
  // whose quotient by W (a row count that may run into the next images) and
  // that row's remainder by H come from multiply-highs.
  const uint32_t rem0 =
      (uint32_t)m0 - div_rcp((uint32_t)m0, (uint32_t)HW, a.rcp_hw) * (uint32_t)HW;
  uint32_t ppix[C::NU], pmask[C::NU], coff[C::NU];
#pragma unroll
  for (int u = 0; u < C::NU; ++u) {
    const int wl = wave + u * C::NW;
    ppix[u] = 0;
    pmask[u] = 0;
    coff[u] = OOB;
    if (u < C::UA) {
      const int r = wl * C::RPL + lane / C::CPR;
      const long m = m0 + r;
      const uint32_t t = rem0 + (uint32_t)r;
      const uint32_t hr = div_rcp(t, (uint32_t)W, a.rcp_w);
      const uint32_t w = t - hr * (uint32_t)W;
      const uint32_t h = hr - div_rcp(hr, (uint32_t)H, a.rcp_h) * (uint32_t)H;
      // taps t = 3 (dy + 1) + dx + 1: rows dy valid in rv, columns dx in cv
      const uint32_t rv = (h > 0 ? 1u : 0u) | 2u | (h + 1 < (uint32_t)H ? 4u : 0u);
      const uint32_t cv = (w > 0 ? 1u : 0u) | 2u | (w + 1 < (uint32_t)W ? 4u : 0u);
      const uint32_t mask = ((rv & 1u) ? cv : 0u) | ((rv & 2u) ? cv << 3 : 0u) |
                            ((rv & 4u) ? cv << 6 : 0u);
      ppix[u] = (uint32_t)(m < P ? m : 0);
      pmask[u] = m < P ? mask : 0u;
      coff[u] = (uint32_t)(((lane % C::CPR) ^ swz_row<C::RB>(r)) * 16);
    } else if (wl < C::WL) {
      const int r = (wl - C::WLA) * C::RPL + lane / C::CPR;
      const int n = n0 + r;
      coff[u] = n < a.N ? (uint32_t)n * (uint32_t)(a.ldb * 2) +
                              (uint32_t)(((lane % C::CPR) ^ swz_row<C::RB>(r)) * 16)
                        : OOB;
    }
  }

  const SegRt q1 = seg_rt(a.seg[1], P);
  const SegRt q2 = seg_rt(a.seg[2], P);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.Bw, (long)a.N * a.ldb * 2);
  const uint32_t sbase = lds_u32(smem);

  // K position of the next stage to issue: segment, channel chunk and tap
  // (dy, dx), walked chunk-major (the taps of one 64-channel chunk run back
  // to back, so the shifted reads of one input slice stay in L2), without
  // divisions.  The weight column of (tap, channel c) is begin + tap*C + c.
  SegRt cur = seg_rt(a.seg[0], P);
  int iseg = 0, itap = 0, icb = 0, idy, idx;
  if (kt0 > 0) {
    int q = kt0;  // first K-step of this split
    while (iseg < 2 && q >= cur.taps * (cur.C / C::BK)) {
      q -= cur.taps * (cur.C / C::BK);
      ++iseg;
      select_into(cur, iseg == 1, q1, q2);
    }
    icb = (q / cur.taps) * C::BK;
    itap = q - (q / cur.taps) * cur.taps;
    idy = cur.taps == 9 ? itap / 3 - 1 : 0;
    idx = cur.taps == 9 ? itap % 3 - 1 : 0;
  } else {
    idy = idx = cur.taps == 9 ? -1 : 0;
  }
  auto advance = [&]() __attribute__((always_inline)) {
    ++itap;
    if (++idx > 1) {
      idx = -1;
      ++idy;
    }
    if (itap >= cur.taps) {
      itap = 0;
      idy = idx = cur.taps == 9 ? -1 : 0;
      icb += C::BK;
      if (icb >= cur.C) {
        icb = 0;
        ++iseg;
        select_into(cur, iseg == 1, q1, q2);
        idy = idx = cur.taps == 9 ? -1 : 0;
      }
    }
  };
  auto issue = [&](uint32_t stage_off) __attribute__((always_inline)) {
    const bool second = icb >= cur.c0;
    const __amdgpu_buffer_rsrc_t rs = second ? cur.r1 : cur.r0;
    const uint32_t pitch = second ? cur.pitch1 : cur.pitch0;
    const uint32_t cbyte = (uint32_t)((second ? icb - cur.c0 : icb) * 2);
    const int t9 = (idy + 1) * 3 + idx + 1;
    const int shift = idy * W + idx;
    const uint32_t kbyte = (uint32_t)((cur.begin + itap * cur.C + icb) * 2);
#pragma unroll
    for (int u = 0; u < C::NU; ++u) {
      const int wl = wave + u * C::NW;
      char* dst = smem + stage_off + wl * 1024;  // 1 KB per wave load
      if (u < C::UA) {
        const uint32_t off = ((pmask[u] >> t9) & 1u)
                                 ? __umul24(ppix[u] + shift, pitch) + cbyte + coff[u]
                                 : OOB;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, lds(dst), 16, off, 0, 0, 0);
      } else if (u < C::NU_LO || wl < C::WL) {
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, lds(dst), 16, coff[u] + kbyte, 0, 0, 0);
      }
    }
    advance();
  };

  f32x4_t acc[C::TM][C::TN];
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // fragment addresses: rows wm*WM + i*16 + r16 (A) and wn*WN + j*16 + r16
  // (B) share one swizzle for every i / j, so each K-half needs one base
  // address per operand and the row step is an immediate offset
  const int r16 = lane & 15;
  const int g4 = lane >> 4;
  uint32_t fa[C::KH], fb[C::KH];
#pragma unroll
  for (int s = 0; s < C::KH; ++s) {
    const int c = s * 4 + g4;
    const int ra = wm * C::WM + r16, rb = wn * C::WN + r16;
    fa[s] = (uint32_t)(ra * C::RB + ((c ^ swz_row<C::RB>(ra)) << 4));
    fb[s] = (uint32_t)(rb * C::RB + ((c ^ swz_row<C::RB>(rb)) << 4));
  }

  // Per K-step: wait for this stage's DMA (the later stages stay in
  // flight), barrier, start the DMA of the stage STAGES-1 ahead into the slot
  // read one step ago, issue every fragment read of this stage, then the
  // MFMAs of each K-half once its fragments have landed.
  bf16x8_t af[C::KH][C::TM], bfr[C::KH][C::TN];
  issue(0);
#pragma unroll
  for (int q = 1; q < C::STAGES - 1; ++q)
    if (q < KT) issue((uint32_t)(q * C::STAGE));
  int slot = 0;
  for (int kt = 0; kt < KT; ++kt) {
    // stages issued after this one: min(STAGES - 2, KT - 1 - kt), each NU
    // (or NU_LO) loads of this wave
    const int after = min(C::STAGES - 2, KT - 1 - kt);
    const bool hi = C::REM == 0 || wave < C::REM;
    if (after <= 0)
      wait_vmcnt<0>();
    else if (after == 1)
      hi ? wait_vmcnt<C::NU>() : wait_vmcnt<C::NU_LO>();
    else
      hi ? wait_vmcnt<2 * C::NU>() : wait_vmcnt<2 * C::NU_LO>();
    __builtin_amdgcn_s_barrier();
    const uint32_t sb = sbase + (uint32_t)(slot * C::STAGE);
    // the slot refilled here was read one step ago: every wave is past that
    if (kt + C::STAGES - 1 < KT) {
      const int ns = slot + C::STAGES - 1;
      issue((uint32_t)((ns >= C::STAGES ? ns - C::STAGES : ns) * C::STAGE));
    }
#pragma unroll
    for (int s = 0; s < C::KH; ++s) {
      ds_rd_n<C::TM, 16 * C::RB, 0>(af[s], sb + fa[s]);
      ds_rd_n<C::TN, 16 * C::RB, C::A_BYTES>(bfr[s], sb + fb[s]);
    }
    slot = slot + 1 == C::STAGES ? 0 : slot + 1;
#pragma unroll
    for (int s = 0; s < C::KH; ++s) {
      // the scheduler must not sink this half's MFMAs below the next
      // half's wait (they would all wait for every fragment read)
      __builtin_amdgcn_sched_barrier(0);
      if (s + 1 < C::KH)
        lgkm_wait<C::TM + C::TN>();
      else
        lgkm_wait<0>();
#pragma unroll
      for (int i = 0; i < C::TM; ++i) tie(af[s][i]);
#pragma unroll
      for (int j = 0; j < C::TN; ++j) tie(bfr[s][j]);
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
          acc[i][j] =
              __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[s][i], bfr[s][j], acc[i][j], 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  __syncthreads();

  // epilogue in 16-row slices: accumulators -> LDS -> 8-channel rows
  // (+bias, +rowvec, +residual) -> 16-byte stores.  With a.stats the stored
  // (bf16-rounded) values go back to the slice in LDS and thread t < BN adds
  // column t of every slice to its running sum and sum of squares: the
  // GroupNorm statistics of the output, one row per (image, M-tile).
  float* ct = reinterpret_cast<float*>(smem);
  constexpr int NV8 = C::BN / 8;
  constexpr int NTK = (16 * NV8 + C::NT - 1) / C::NT;  // tasks per thread and slice
  static_assert(C::BN <= C::NT, "one thread per output column for the statistics");
  const bool stats = !GNB && a.stats != nullptr;
  const bool raw = !GNB && a.ksplit > 1;  // raw partial; the finalize adds the epilogue terms
  const bool has_res = !GNB && a.resid.s0.ptr != nullptr;
  const float* const bias = GNB ? nullptr : a.bias;
  const float* const rowvec = GNB ? nullptr : a.rowvec;
  void* const out2 = GNB ? nullptr : a.out2;
  // A thread's tasks keep their row within a slice and their 8 columns in
  // every slice: the bias and, for a tile inside one image, its timestep
  // row are loaded once; each slice's residual is loaded a slice ahead.
  const long mlast = (m0 + C::BM < P ? m0 + C::BM : P) - 1;
  const int img0 = (int)div_rcp((uint32_t)m0, (uint32_t)HW, a.rcp_hw);
  const bool uni = (int)div_rcp((uint32_t)mlast, (uint32_t)HW, a.rcp_hw) == img0;
  int trow[NTK], tnc[NTK];
  bool tok[NTK];
  float cb[NTK][8], cr[NTK][8], rres[NTK][8];
#pragma unroll
  for (int k = 0; k < NTK; ++k) {
    const int e = tid + k * C::NT;
    trow[k] = e / NV8;
    tnc[k] = n0 + (e - trow[k] * NV8) * 8;
    tok[k] = e < 16 * NV8 && tnc[k] < a.N;
#pragma unroll
    for (int q = 0; q < 8; ++q) cb[k][q] = cr[k][q] = rres[k][q] = 0.f;
    if (tok[k] && !raw) {
      if (bias) {
#pragma unroll
        for (int q = 0; q < 8; ++q) cb[k][q] = bias[tnc[k] + q];
      }
      if (rowvec && uni) {
#pragma unroll
        for (int q = 0; q < 8; ++q) cr[k][q] = rowvec[(long)img0 * a.N + tnc[k] + q];
      }
    }
  }
  auto load_res = [&](int g, int i) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < NTK; ++k) {
      const long m = m0 + g * C::WM + i * 16 + trow[k];
      if (tok[k] && m < P) ld8(a.resid.s0, m, tnc[k], rres[k]);
    }
  };
  if (has_res && !raw) load_res(0, 0);
  float csum = 0.f, csq = 0.f;
  // GroupNorm-backward sums (a.gnb; whole tiles inside image img0, no K
  // split).  The folded per-channel constants of the tile's columns sit in
  // LDS after the staging slice (scale, shift, rstd, -mean * rstd); each
  // slice's dz and dz * xhat go to LDS and thread t < BN adds column t over
  // the slice's rows, as for the output statistics.  x of the next slice is
  // in flight while the current one is processed.
  constexpr bool gnb = GNB;
  float* gk = ct + 2 * 16 * C::LDC;  // [4][BN]
  uint4 gxr[NTK];
#pragma unroll
  for (int k = 0; k < NTK; ++k) gxr[k] = uint4{0u, 0u, 0u, 0u};
  auto load_gx = [&](int g, int i) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < NTK; ++k) {
      const long m = m0 + g * C::WM + i * 16 + trow[k];
      if (tok[k] && m < P) {
        const VIn& x = a.gnb_x;
        const int c = tnc[k];
        const Src& sx = c < x.c0 ? x.s0 : x.s1;
        gxr[k] = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(sx.ptr) + m * sx.C +
                                                 (c < x.c0 ? c : c - x.c0));
      }
    }
  };
  float gsz = 0.f, gsx = 0.f;
  if (gnb) {
    load_gx(0, 0);
    if (tid < C::BN && n0 + tid < a.N) {
      const int c = n0 + tid;
      const int gi = img0 * a.gnb_G + c / (a.N / a.gnb_G);
      const float rs = a.gnb_rstd[gi];
      gk[tid] = a.gnb_scale[(long)img0 * a.N + c];
      gk[C::BN + tid] = a.gnb_shift[(long)img0 * a.N + c];
      gk[2 * C::BN + tid] = rs;
      gk[3 * C::BN + tid] = -a.gnb_mean[gi] * rs;
    }
  }
#pragma unroll 1
  for (int g = 0; g < C::WAVES_M; ++g) {
#pragma unroll
    for (int i = 0; i < C::TM; ++i) {
      if (wm == g) acc16_to_lds<C::TM, C::TN, C::WN, C::LDC>(ct, wn, lane, i, acc);
      __syncthreads();
      float rcur[NTK][8];
#pragma unroll
      for (int k = 0; k < NTK; ++k)
#pragma unroll
        for (int q = 0; q < 8; ++q) rcur[k][q] = rres[k][q];
      if (has_res && !raw) {
        if (i + 1 < C::TM)
          load_res(g, i + 1);
        else if (g + 1 < C::WAVES_M)
          load_res(g + 1, 0);
      }
      uint4 xcur[NTK];
#pragma unroll
      for (int k = 0; k < NTK; ++k) xcur[k] = gxr[k];
      if (gnb) {
        if (i + 1 < C::TM)
          load_gx(g, i + 1);
        else if (g + 1 < C::WAVES_M)
          load_gx(g + 1, 0);
      }
#pragma unroll
      for (int k = 0; k < NTK; ++k) {
        const int row = trow[k];
        const int n = tnc[k];
        const long m = m0 + g * C::WM + i * 16 + row;
        if (!tok[k] || m >= P) continue;
        float* src = ct + row * C::LDC + (n - n0);
        const float4 s0 = reinterpret_cast<const float4*>(src)[0];
        const float4 s1 = reinterpret_cast<const float4*>(src)[1];
        if (raw) {
          float4* dp = reinterpret_cast<float4*>(a.part + ((long)z * P + m) * a.N + n);
          dp[0] = s0;
          dp[1] = s1;
          continue;
        }
        float v[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
        if (bias) {
#pragma unroll
          for (int q = 0; q < 8; ++q) v[q] += cb[k][q];
        }
        if (rowvec) {
          if (uni) {
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] += cr[k][q];
          } else {
            const float* rv = rowvec + (long)(m / HW) * a.N + n;
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] += rv[q];
          }
        }
        if (has_res) {
#pragma unroll
          for (int q = 0; q < 8; ++q) v[q] += rcur[k][q];
        }
        st8(a.out, a.out_dtype, a.ldo, m, n, v);
        if (out2) st8(out2, a.out_dtype, a.ldo, m, n, v);
        if (gnb) {
          // da as stored (the separate backward pass reads the bf16 tensor);
          // dz to the staging slice, dz * xhat to the one after it
          const uint32_t xw[4] = {xcur[k].x, xcur[k].y, xcur[k].z, xcur[k].w};
          const float* kc = gk + (n - n0);
          float dzv[8], dxv[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const float x = __uint_as_float(q & 1 ? xw[q / 2] & 0xffff0000u : xw[q / 2] << 16);
            const float d = a.out_dtype == DT_BF16 ? bf2f(f2bf(v[q])) : v[q];
            const float dz = d * dsilu_f(x * kc[q] + kc[C::BN + q]);
            dzv[q] = dz;
            dxv[q] = dz * (x * kc[2 * C::BN + q] + kc[3 * C::BN + q]);
          }
          float4* w = reinterpret_cast<float4*>(src);
          w[0] = make_float4(dzv[0], dzv[1], dzv[2], dzv[3]);
          w[1] = make_float4(dzv[4], dzv[5], dzv[6], dzv[7]);
          float4* w2 = reinterpret_cast<float4*>(src + 16 * C::LDC);
          w2[0] = make_float4(dxv[0], dxv[1], dxv[2], dxv[3]);
          w2[1] = make_float4(dxv[4], dxv[5], dxv[6], dxv[7]);
        }
        if (stats) {
          float4* w = reinterpret_cast<float4*>(src);
          w[0] = make_float4(bf2f(f2bf(v[0])), bf2f(f2bf(v[1])), bf2f(f2bf(v[2])),
                             bf2f(f2bf(v[3])));
          w[1] = make_float4(bf2f(f2bf(v[4])), bf2f(f2bf(v[5])), bf2f(f2bf(v[6])),
                             bf2f(f2bf(v[7])));
        }
      }
      __syncthreads();
      if (stats) {
        if (tid < C::BN) {
#pragma unroll 4
          for (int row = 0; row < 16; ++row) {
            const float x = ct[row * C::LDC + tid];
            csum += x;
            csq += x * x;
          }
        }
        __syncthreads();
      }
      if (gnb) {
        // rows past P hold no task's values: only whole tiles take this path
        if (tid < C::BN) {
#pragma unroll 4
          for (int row = 0; row < 16; ++row) {
            gsz += ct[row * C::LDC + tid];
            gsx += ct[(16 + row) * C::LDC + tid];
          }
        }
        __syncthreads();
      }
    }
  }
  if (stats && tid < C::BN && n0 + tid < a.N) {
    const int img = img0;
    const int chunk = (int)(m0 - (long)img * HW) / C::BM;
    float* dst = a.stats + ((long)img * (HW / C::BM) + chunk) * 2 * a.N + n0 + tid;
    dst[0] = csum;
    dst[a.N] = csq;
  }
  if (gnb && tid < C::BN && n0 + tid < a.N) {
    const int chunk = (int)(m0 - (long)img0 * HW) / C::BM;
    float* dst = a.gnb + ((long)img0 * (HW / C::BM) + chunk) * 2 * a.N + n0 + tid;
    dst[0] = gsz;
    dst[a.N] = gsx;
  }
#else
  (void)a;
#endif
}

// ---------------------------------------------------------------------------
// WGRAD mode
// ---------------------------------------------------------------------------

template <class C>
__global__ __launch_bounds__(C::NT) void igemm2_wgrad(GemmArgs a, const void* zero16) {
  // the body exists for the device pass only (the host pass emits the launch stub)
#if defined(__HIP_DEVICE_COMPILE__)
  __shared__ __attribute__((aligned(1024))) char smem[2 * C::STAGE];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar registers
  const int wm = wave % C::WAVES_M;
  const int wn = wave / C::WAVES_M;

  // block -> (pixel split z, tile), split-major over a contiguous range per
  // XCD, so the blocks of one pixel split share that XCD's L2; split z
  // covers kchunk pixels
  const int tilesN = (a.N + C::BN - 1) / C::BN;
  const int ntiles = ((a.M + C::BM - 1) / C::BM) * tilesN;
  const int lb = xcd_remap(blockIdx.x, gridDim.x);
  const int H = a.g.H, W = a.g.W, HW = a.g.H * a.g.W;
  const long P = a.g.pixels();
  const int z = (int)div_rcp((uint32_t)lb, (uint32_t)ntiles, a.rcp_nt);
  const int tile = lb - z * ntiles;
  const long pbeg = (long)z * a.kchunk;
  const long pend = (pbeg + a.kchunk < P) ? pbeg + a.kchunk : P;
  const int tmi = (int)div_rcp((uint32_t)tile, (uint32_t)tilesN, a.rcp_tn);
  const int m0 = tmi * C::BM;
  const int n0 = (tile - tmi * tilesN) * C::BN;

  const __amdgpu_buffer_rsrc_t rg = make_rsrc(a.gy.s0.ptr, P * a.gy.s0.C * 2);
  const uint32_t gpitch = (uint32_t)(a.gy.s0.C * 2);

  // Per wave load u: A loads (wl < WLA) fetch dY rows; B loads fetch the
  // shifted activation columns through per-lane addresses.  Lane slot q of
  // a load is physical chunk q % C of pixel row q / C; it fetches the
  // logical chunk the row's rotation puts there.
  int rrow[C::NU];          // pixel row of the tile
  uint32_t aoff[C::NU];     // A: channel byte offset in dY, or OOB
  const char* bsrc[C::NU];  // B: source pointer at the column's channel
  uint32_t bpitch[C::NU];
  int bshift[C::NU], boy[C::NU], box[C::NU];
  int bh[C::NU], bw[C::NU];  // B: image row / column of the current pixel
#pragma unroll
  for (int u = 0; u < C::NU; ++u) {
    const int wl = wave + u * C::NW;
    bsrc[u] = nullptr;
    bpitch[u] = 0;
    bshift[u] = boy[u] = box[u] = bh[u] = bw[u] = 0;
    aoff[u] = OOB;
    if (u < C::UA) {
      const int q = wl * 64 + lane;
      const int r = q / C::CA;
      const int lc = rot_logical(q - r * C::CA, r, C::CA, C::RA_A, C::RA_B);
      rrow[u] = r;
      const int o = m0 + lc * 8;
      aoff[u] = o < a.M ? (uint32_t)(o * 2) : OOB;
    } else {
      const int q = (wl - C::WLA) * 64 + lane;
      const int r = q / C::CB;
      const int lc = rot_logical(q - r * C::CB, r, C::CB, C::RB_A, C::RB_B);
      rrow[u] = r;
      const int n = n0 + lc * 8;
      if (n < a.N) {
        const int s = seg_of(a.nseg, a.seg[1].begin, a.seg[2].begin, n);
        const Seg& sg = s == 0 ? a.seg[0] : (s == 1 ? a.seg[1] : a.seg[2]);
        const int rr = n - sg.begin;
        const uint32_t rc = s == 0 ? a.rcp_segc[0] : (s == 1 ? a.rcp_segc[1] : a.rcp_segc[2]);
        const int tap = (int)div_rcp((uint32_t)rr, (uint32_t)sg.C, rc);
        const int c = rr - tap * sg.C;
        const int t9 = sg.taps == 9 ? tap : 4;
        boy[u] = t9 / 3 - 1;
        box[u] = t9 % 3 - 1;
        bshift[u] = boy[u] * W + box[u];
        const bool second = c >= sg.in.c0;
        const Src& src = second ? sg.in.s1 : sg.in.s0;
        bsrc[u] = static_cast<const char*>(src.ptr) + (second ? c - sg.in.c0 : c) * 2;
        bpitch[u] = (uint32_t)(src.C * 2);
      }
      // image coordinates of pixel pbeg + r (advanced by 64 per K-step)
      const long p = pbeg + r;
      const long pp = p < P ? p : 0;
      const uint32_t img = div_rcp((uint32_t)pp, (uint32_t)HW, a.rcp_hw);
      const uint32_t rem = (uint32_t)pp - img * (uint32_t)HW;
      const uint32_t hq = div_rcp(rem, (uint32_t)W, a.rcp_w);
      bh[u] = (int)hq;
      bw[u] = (int)(rem - hq * (uint32_t)W);
    }
  }

  // one K-step of BK pixels moves a pixel by kdw columns and kdh rows
  // (kdh < H; the carry of the columns adds at most one more row)
  const int kq = (int)div_rcp((uint32_t)C::BK, (uint32_t)W, a.rcp_w);
  const int kdw = C::BK - kq * W;
  const int kdh = kq - (int)div_rcp((uint32_t)kq, (uint32_t)H, a.rcp_h) * H;
  auto issue = [&](int kt, char* base) __attribute__((always_inline)) {
    const long p0 = pbeg + (long)kt * C::BK;
#pragma unroll
    for (int u = 0; u < C::NU; ++u) {
      const int wl = wave + u * C::NW;
      const long p = p0 + rrow[u];
      if (u < C::UA) {
        const uint32_t off = p < pend ? (uint32_t)p * gpitch + aoff[u] : OOB;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rg, lds(base + wl * 1024), 16, off, 0, 0, 0);
      } else {
        const int hh = bh[u] + boy[u], ww = bw[u] + box[u];
        const bool ok = bsrc[u] && p < pend && hh >= 0 && hh < H && ww >= 0 && ww < W;
        const void* g = ok ? (const void*)(bsrc[u] + (long)(p + bshift[u]) * bpitch[u]) : zero16;
        __builtin_amdgcn_global_load_lds(g, lds(base + C::A_BYTES + (wl - C::WLA) * 1024), 16, 0,
                                         0);
        // advance this lane's pixel by one K-step: BK = kdh rows + kdw
        // columns, the row taken modulo H (the next image starts at row 0)
        int w = bw[u] + kdw, h = bh[u] + kdh;
        if (w >= W) {
          w -= W;
          ++h;
        }
        if (h >= H) h -= H;
        bw[u] = w;
        bh[u] = h;
      }
    }
  };

  f32x4_t acc[C::TM][C::TN];
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Transpose reads: lane (g16, j16) addresses pixel row
  // trow = 8 g16 + j16 / 4 (+ 32 s + 4 h) and channel 4 (j16 % 4) of a
  // fragment's 16 columns.  Row bits 0-1 and 3 are fixed per lane, so the
  // rotation and hence each fragment's column byte offset is too; the row
  // step (s, h) is an immediate.
  const int g16 = lane >> 4;
  const int j16 = lane & 15;
  const int trow = 8 * g16 + (j16 >> 2);
  const int tcol = 4 * (j16 & 3);
  uint32_t ra[C::TM], rb[C::TN];
#pragma unroll
  for (int i = 0; i < C::TM; ++i) {
    const int col = wm * C::WM + i * 16 + tcol;
    ra[i] = (uint32_t)(trow * C::PA + rot_slot(col >> 3, trow, C::CA, C::RA_A, C::RA_B) * 16 +
                       (col & 7) * 2);
  }
#pragma unroll
  for (int j = 0; j < C::TN; ++j) {
    const int col = wn * C::WN + j * 16 + tcol;
    rb[j] = (uint32_t)(trow * C::PB + rot_slot(col >> 3, trow, C::CB, C::RB_A, C::RB_B) * 16 +
                       (col & 7) * 2);
  }
  const uint32_t sbase = lds_u32(smem);

  bf16x8_t af[2][C::TM], bfr[2][C::TN];
  auto read = [&](uint32_t sb, bf16x8_t (&fa)[C::TM], bf16x8_t (&fb)[C::TN], auto s_tag)
      __attribute__((always_inline)) {
    constexpr int S = decltype(s_tag)::value;
#pragma unroll
    for (int i = 0; i < C::TM; ++i) {
      const v4s lo = ds_rdtr<(S * 32 + 0) * C::PA>(sb + ra[i]);
      const v4s hi = ds_rdtr<(S * 32 + 4) * C::PA>(sb + ra[i]);
      fa[i] = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    }
#pragma unroll
    for (int j = 0; j < C::TN; ++j) {
      const v4s lo = ds_rdtr<C::A_BYTES + (S * 32 + 0) * C::PB>(sb + rb[j]);
      const v4s hi = ds_rdtr<C::A_BYTES + (S * 32 + 4) * C::PB>(sb + rb[j]);
      fb[j] = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    }
  };
  auto mma = [&](bf16x8_t (&fa)[C::TM], bf16x8_t (&fb)[C::TN]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < C::TM; ++i) tie(fa[i]);
#pragma unroll
    for (int j = 0; j < C::TN; ++j) tie(fb[j]);
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
      for (int j = 0; j < C::TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
  };

  // Per K-step: wait for the stage, barrier, read the first 32 pixels'
  // fragments, start the next stage's DMA, then the second half's reads
  // overlap the first half's MFMAs.
  const int KT = (int)((pend - pbeg + C::BK - 1) / C::BK);
  if (KT > 0) issue(0, smem);
  for (int kt = 0; kt < KT; ++kt) {
    wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    const uint32_t sb = sbase + (uint32_t)((kt & 1) * C::STAGE);
    read(sb, af[0], bfr[0], std::integral_constant<int, 0>());
    if (kt + 1 < KT) issue(kt + 1, smem + ((kt + 1) & 1) * C::STAGE);
    lgkm_wait<0>();
    read(sb, af[1], bfr[1], std::integral_constant<int, 1>());
    mma(af[0], bfr[0]);
    // keep the first half's MFMAs above the second half's wait
    __builtin_amdgcn_sched_barrier(0);
    lgkm_wait<0>();
    mma(af[1], bfr[1]);
    __builtin_amdgcn_sched_barrier(0);
  }
  __syncthreads();

  // fp32 partials through LDS, GPP wave rows (GPP * WM tile rows) at a
  // time: those waves stage all their accumulators, then every thread
  // stores 16-byte row pieces, into the split's partial or, with one pixel
  // split, added into the gradient (one writer per element)
  float* ct = reinterpret_cast<float*>(smem);
  float* part = a.part + (long)z * a.M * a.N;
  constexpr int NV4 = C::BN / 4;
  constexpr int GPP = (2 * C::STAGE) / (C::WM * C::LDC * 4);  // wave rows per pass
  static_assert(GPP >= 1, "one wave row of accumulators fits the LDS stages");
  constexpr int ROWS = (GPP < C::WAVES_M ? GPP : C::WAVES_M) * C::WM;
  constexpr int IT = (ROWS * NV4 + C::NT - 1) / C::NT;  // row pieces per thread and pass
#pragma unroll 1
  for (int g0 = 0; g0 < C::WAVES_M; g0 += GPP) {
    // one pixel split: fetch this pass's gradient pieces before staging the
    // accumulators, so that their loads are in flight together (the host
    // guarantees 16-byte aligned rows of a multiple of 4 columns)
    float4 gv[IT];
    float* gp[IT];
    if (a.wdirect) {
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const int e = tid + it * C::NT;
        const int row = e / NV4;
        const int n = n0 + (e - row * NV4) * 4;
        const int m = m0 + g0 * C::WM + row;
        gp[it] = nullptr;
        gv[it] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (e >= ROWS * NV4 || row >= (C::WAVES_M - g0) * C::WM || m >= a.M || n >= a.N)
          continue;
        // segment bounds are multiples of 8: the four columns share one
        const int s = seg_of(a.nseg, a.seg[1].begin, a.seg[2].begin, n);
        const Seg& sg = s == 0 ? a.seg[0] : (s == 1 ? a.seg[1] : a.seg[2]);
        gp[it] = sg.grad + (long)m * (sg.end - sg.begin) + (n - sg.begin);
        gv[it] = *reinterpret_cast<const float4*>(gp[it]);
      }
    }
    if (wm >= g0 && wm < g0 + GPP) {
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
        acc16_to_lds<C::TM, C::TN, C::WN, C::LDC>(ct + ((wm - g0) * C::WM + i * 16) * C::LDC, wn,
                                                  lane, i, acc);
    }
    __syncthreads();
    if (a.wdirect) {
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        if (!gp[it]) continue;
        const int e = tid + it * C::NT;
        const int row = e / NV4;
        const int c = (e - row * NV4) * 4;
        const float4 v = *reinterpret_cast<const float4*>(ct + row * C::LDC + c);
        const float4 g = gv[it];
        *reinterpret_cast<float4*>(gp[it]) =
            make_float4(g.x + v.x, g.y + v.y, g.z + v.z, g.w + v.w);
      }
    } else {
      for (int e = tid; e < ROWS * NV4; e += C::NT) {
        const int row = e / NV4;
        const int n = n0 + (e - row * NV4) * 4;
        const int m = m0 + g0 * C::WM + row;
        if (row >= (C::WAVES_M - g0) * C::WM || m >= a.M || n >= a.N) continue;
        *reinterpret_cast<float4*>(part + (long)m * a.N + n) =
            *reinterpret_cast<const float4*>(ct + row * C::LDC + (n - n0));
      }
    }
    __syncthreads();
  }
#else
  (void)a;
  (void)zero16;
#endif
}

// ---------------------------------------------------------------------------
// K-split conv finalize: out = sum_z part[z] (fixed order) + bias + rowvec +
// residual, one 8-channel vector per thread
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void conv_splitk_finalize(GemmArgs a) {
  const long P = a.g.pixels();
  const int NV = a.N / 8;
  const int HW = a.g.H * a.g.W;
  const long total = P * NV;
  const long zs = P * a.N;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (long)gridDim.x * blockDim.x) {
    const long m = i / NV;
    const int n = (int)(i - m * NV) * 8;
    const float* src = a.part + m * a.N + n;
    float v[8];
    {
      const float4 s0 = reinterpret_cast<const float4*>(src)[0];
      const float4 s1 = reinterpret_cast<const float4*>(src)[1];
      v[0] = s0.x; v[1] = s0.y; v[2] = s0.z; v[3] = s0.w;
      v[4] = s1.x; v[5] = s1.y; v[6] = s1.z; v[7] = s1.w;
    }
    for (int zz = 1; zz < a.ksplit; ++zz) {
      const float4 s0 = reinterpret_cast<const float4*>(src + zz * zs)[0];
      const float4 s1 = reinterpret_cast<const float4*>(src + zz * zs)[1];
      v[0] += s0.x; v[1] += s0.y; v[2] += s0.z; v[3] += s0.w;
      v[4] += s1.x; v[5] += s1.y; v[6] += s1.z; v[7] += s1.w;
    }
    if (a.bias) {
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] += a.bias[n + q];
    }
    if (a.rowvec) {
      const float* rv = a.rowvec + (m / HW) * a.N + n;
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] += rv[q];
    }
    if (a.resid.s0.ptr) {
      float rr[8];
      ld8(a.resid.s0, m, n, rr);
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] += rr[q];
    }
    st8(a.out, a.out_dtype, a.ldo, m, n, v);
    if (a.out2) st8(a.out2, a.out_dtype, a.ldo, m, n, v);
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

namespace launch2 {
using C2_128x160 = CfgC<128, 160, 64, 80>;   // 4 waves, two blocks per CU
using C2_128x128 = CfgC<128, 128, 64, 64>;   // 4 waves, two blocks per CU
using C2_128x192 = CfgC<128, 192, 64, 96>;   // 4 waves, two blocks per CU
using C2_64x128S3 = CfgC<64, 128, 32, 64, 3>;  // 4 waves, 3 stages, two blocks per CU
using W2_320x128 = CfgW<320, 128, 80, 64>;   // 8 waves, one block per CU
using W2_128x128 = CfgW<128, 128, 64, 64>;   // 4 waves

template <class C>
static hipError_t conv2_t(const GemmArgs& a_in, hipStream_t st, hipEvent_t t0, hipEvent_t t1) {
  // 32-bit pixel indices and weight offsets
  if (a_in.g.pixels() + C::BM >= (1L << 31) || (long)a_in.N * a_in.ldb * 2 >= (1L << 31))
    return hipErrorInvalidValue;
  GemmArgs a = a_in;
  {
    const long P = a.g.pixels(), HW = a.g.hw();
    const long tN = (a.N + C::BN - 1) / C::BN, nt = ((P + C::BM - 1) / C::BM) * tN;
    const long ks = a.ksplit > 1 ? a.ksplit : 1;
    a.rcp_nt = rcp_u32(nt, nt * ks);
    a.rcp_tn = rcp_u32(tN, nt);
    a.rcp_hw = rcp_u32(HW, P + C::BM);
    a.rcp_w = rcp_u32(a.g.W, HW + C::BM);
    a.rcp_h = rcp_u32(a.g.H, (HW + C::BM) / a.g.W + 1);
  }
  // output statistics need whole tiles inside one image and no K split
  if ((a.stats || a.gnb) && (a.ksplit > 1 || a.g.hw() % C::BM != 0)) return hipErrorInvalidValue;
  if (a.gnb && (a.gnb_G < 1 || a.N % a.gnb_G != 0 || a.resid.s0.ptr || a.bias || a.rowvec ||
                a.out2 || a.stats || a.out_dtype != DT_BF16 || a.gnb_x.s0.dtype != DT_BF16 ||
                (a.gnb_x.c0 < a.gnb_x.C && a.gnb_x.s1.dtype != DT_BF16) || a.gnb_x.add))
    return hipErrorInvalidValue;
  const long tilesM = (a.g.pixels() + C::BM - 1) / C::BM;
  const long tilesN = (a.N + C::BN - 1) / C::BN;
  const int ks = a.ksplit > 1 ? a.ksplit : 1;
  const bool fin = ks > 1 && !a.skip_finalize;  // the K-split finalize follows here
  const dim3 grid((unsigned)(tilesM * tilesN * ks)), block(C::NT);
  auto kern = a.gnb ? igemm2_conv<C, true> : igemm2_conv<C, false>;
  if (t0 || t1)
    hipExtLaunchKernelGGL(kern, grid, block, 0, st, t0, fin ? nullptr : t1, 0, a);
  else
    hipLaunchKernelGGL(kern, grid, block, 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !fin) return e;
  const long vec = a.g.pixels() * (a.N / 8);
  const long blocks = std::min<long>((vec + 255) / 256, 2048);
  if (t1)
    hipExtLaunchKernelGGL(conv_splitk_finalize, dim3((unsigned)blocks), dim3(256), 0, st, nullptr,
                          t1, 0, a);
  else
    hipLaunchKernelGGL(conv_splitk_finalize, dim3((unsigned)blocks), dim3(256), 0, st, a);
  return hipGetLastError();
}

// One pixel split with 16-byte aligned gradient rows of a multiple of 4
// columns: the GEMM epilogue adds into the gradients and no finalize runs.
static bool wgrad_direct(const GemmArgs& a, int splits) {
  if (splits != 1) return false;
  for (int i = 0; i < a.nseg; ++i)
    if (reinterpret_cast<uintptr_t>(a.seg[i].grad) % 16 != 0 ||
        (a.seg[i].end - a.seg[i].begin) % 4 != 0)
      return false;
  return true;
}

template <class C>
static hipError_t wgrad2_t(const GemmArgs& a_in, int splits, const void* zero16, hipStream_t st) {
  if (a_in.g.pixels() >= (1L << 31)) return hipErrorInvalidValue;  // 32-bit pixel indices
  GemmArgs a = a_in;
  const long tilesM = (a.M + C::BM - 1) / C::BM;
  const long tilesN = (a.N + C::BN - 1) / C::BN;
  const long blocks = tilesM * tilesN * splits;
  a.wdirect = wgrad_direct(a, splits);
  {
    const long HW = a.g.hw();
    a.rcp_nt = rcp_u32(tilesM * tilesN, blocks);
    a.rcp_tn = rcp_u32(tilesN, tilesM * tilesN);
    a.rcp_hw = rcp_u32(HW, a.g.pixels());
    a.rcp_w = rcp_u32(a.g.W, std::max<long>(HW, C::BK));
    a.rcp_h = rcp_u32(a.g.H, C::BK);
    for (int i = 0; i < a.nseg && i < 3; ++i)
      a.rcp_segc[i] = rcp_u32(a.seg[i].C, (long)a.seg[i].taps * a.seg[i].C);
  }
  hipLaunchKernelGGL(igemm2_wgrad<C>, dim3((unsigned)blocks), dim3(C::NT), 0, st, a, zero16);
  return hipGetLastError();
}

template <class C>
static TileInfo info2() {
  constexpr int lds = C::LDS_BYTES;
  return TileInfo{C::BM, C::BN, C::BK, (160 * 1024) / lds};
}
}  // namespace launch2
using namespace launch2;

TileInfo tile2_info(int t) {
  switch (t) {
    case TILE2_C128x160: return info2<C2_128x160>();
    case TILE2_C128x128: return info2<C2_128x128>();
    case TILE2_C128x192: return info2<C2_128x192>();
    case TILE2_C64x128S3: return info2<C2_64x128S3>();
    case TILE2_W320x128: return info2<W2_320x128>();
    default: return info2<W2_128x128>();
  }
}

hipError_t launch_conv2(const GemmArgs& a, int t, hipStream_t st, hipEvent_t t0, hipEvent_t t1) {
  switch (t) {
    case TILE2_C128x160: return conv2_t<C2_128x160>(a, st, t0, t1);
    case TILE2_C128x192: return conv2_t<C2_128x192>(a, st, t0, t1);
    case TILE2_C64x128S3: return conv2_t<C2_64x128S3>(a, st, t0, t1);
    default: return conv2_t<C2_128x128>(a, st, t0, t1);
  }
}

hipError_t launch_wgrad2(const GemmArgs& a, int t, int splits, const void* zero16,
                         hipStream_t st) {
  hipError_t e;
  switch (t) {
    case TILE2_W320x128: e = wgrad2_t<W2_320x128>(a, splits, zero16, st); break;
    default: e = wgrad2_t<W2_128x128>(a, splits, zero16, st); break;
  }
  if (e != hipSuccess || wgrad_direct(a, splits)) return e;  // added in the epilogue
  return launch_wgrad_finalize(a, splits, st);
}

}  // namespace pulse
