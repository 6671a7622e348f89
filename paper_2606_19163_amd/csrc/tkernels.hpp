// Internal launcher interface of the transformer-block kernels (attn.hip,
// tnorm.hip).  Activations are token-major [T][C] bf16; not part of the
// public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pulse {

// ---- multi-head attention (attn.hip) -------------------------------------

// Head dimension 64, L % 64 == 0, 64 <= L <= ATTN_LMAX, C == heads * 64.
// Up to 256 tokens a head's keys and values sit in LDS whole; longer
// sequences stream them in 64-token chunks (online softmax in the forward).
constexpr int ATTN_LMAX = 4096;
bool attn_fits(int L, int C, int heads);
// o[b*L + i][64 h + e] = sum_j p[b][h][i][j] v[b*L + j][64 h + e] with
// p = softmax_j(q_i . k_j / 8); q, k, v are channel thirds of qkv [B*L][3C].
// lse [B][heads][L] receives log sum_j exp(q_i . k_j / 8) (fp32).
hipError_t launch_attn_fwd(const void* qkv, int B, int L, int C, int heads, void* o, float* lse,
                           hipStream_t st);
// dqkv [B*L][3C] from dout [B*L][C], the forward's o and lse and qkv; dsum
// [B][heads][L] (fp32) is scratch (receives rowsum(dout o)).
hipError_t launch_attn_bwd(const void* qkv, const void* o, const void* dout, const float* lse,
                           int B, int L, int C, int heads, void* dqkv, float* dsum,
                           hipStream_t st);

// ---- LayerNorm, GELU (tnorm.hip) -----------------------------------

// C % 8 == 0 and C <= 2048.
// y = LN(x) * g + b per token; stats[2 t] = mean, stats[2 t + 1] = rstd.
hipError_t launch_ln_fwd(const void* x, long T, int C, float eps, const float* g, const float* b,
                         void* y, float* stats, hipStream_t st);
// dx = add + d LN / dx (add [T][C] bf16 or null); part[ln_bwd_blocks(T)][2][C]
// receives per-block sums of dy * xhat (row 0) and dy (row 1); csum (or
// null), [ln_bwd_blocks(T)][2][C], per-block column sums of dx as stored in
// row 0.
int ln_bwd_blocks(long T);
hipError_t launch_ln_bwd(const void* dy, const void* x, const float* stats, const float* g,
                         const void* add, long T, int C, void* dx, float* part, float* csum,
                         hipStream_t st);

// m = GELU(z) (erf form), n % 8 == 0 elements
hipError_t launch_gelu_fwd(const void* z, void* m, long n, hipStream_t st);
// dz = dm * GELU'(z); dz may alias dm
hipError_t launch_gelu_bwd(const void* dm, const void* z, void* dz, long n, hipStream_t st);

}  // namespace pulse
