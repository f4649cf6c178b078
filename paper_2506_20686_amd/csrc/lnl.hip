// Fused layer-norm + linear projection (MegaFold Section IV, "fused
// layer-norm & linear projection"; forward and backward formulas in the
// appendix table of fused operators), the step that turns the pair
// representation into the triangle-attention inputs:
//   o1 = (x - mean) rstd * gamma + beta   per row of x [M][K],
//   o2 = o1 W                             (W [K][N], no bias),
// with o2's columns written into n_out separate row-major tensors (for the
// attention: Q, K, V, G and the bias logits), so no split copy follows.
//
// Differences from the paper's two-kernel Triton design, for gfx950:
//  - K = 128 (the pair channel width) fits one wave's registers, so the row
//    statistics are computed inside the projection kernel (no separate
//    mean/var pass): a lane holds half a row, two passes over registers give
//    mean and the biased variance, and the normalised row goes straight into
//    the MFMA operand registers in bf16;
//  - the product is formed transposed, o2^T = W^T o1^T (lane <-> row), so
//    each lane stores runs of four consecutive output columns of its row;
//  - the backward's sums over rows (dW, dgamma, dbeta) go to per-block
//    partial sums reduced in a fixed order instead of atomics.
#include "kernels.h"
#include "timing.h"

namespace triattn {

// ---- forward --------------------------------------------------------------------------

// W [K][N] -> W^T [np][K] (rows n >= N are zero): the A operand of o2^T =
// W^T o1^T reads 16 contiguous bytes of a W^T row per lane.
__global__ __launch_bounds__(256) void lnl_wt_kernel(const bf16* w, int N, int np, bf16* wt) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)np * LNL_K) return;
  const int n = (int)(idx / LNL_K), k = (int)(idx % LNL_K);
  wt[idx] = n < N ? w[(int64_t)k * N + n] : (bf16)0.f;
}

// One wave = 32 rows (lane <-> row, lane half g holds features 16 t + 8 g ..
// + 7 for t = 0..7).  Workgroup = 4 waves = 128 rows.
__global__ __launch_bounds__(256) void lnl_fwd_kernel(LnlArgs a) {
  using M = Mma<bf16>;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int wave = tid >> 6;
  const int64_t m = (int64_t)blockIdx.x * 128 + wave * 32 + l32;
  const bool mok = m < a.m;
  constexpr int NT = LNL_K / 16;  // MFMA contraction steps over the features

  bf16x8 xr[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
    xr[t] = mok ? *(const bf16x8*)(a.x + m * LNL_K + 16 * t + 8 * g) : bf16x8{};
  // row statistics: this lane's 64 features, then the other half (lane ^ 32)
  float s = 0.f;
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int e = 0; e < 8; ++e) s += (float)xr[t][e];
  const float mean = wave_xor32_sum(s) * (1.f / LNL_K);
  float v = 0.f;
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float c = (float)xr[t][e] - mean;
      v += c * c;
    }
  const float var = wave_xor32_sum(v) * (1.f / LNL_K);
  const float rstd = 1.f / sqrtf(var + a.eps);
  if (mok && g == 0) {
    a.mean[m] = mean;
    a.rstd[m] = rstd;
  }
  // o1 = xhat gamma + beta as the B operand (contraction over the features)
  bf16x8 of[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const bf16x8 gm = *(const bf16x8*)(a.gamma + 16 * t + 8 * g);
    const bf16x8 bt = *(const bf16x8*)(a.beta + 16 * t + 8 * g);
#pragma unroll
    for (int e = 0; e < 8; ++e)
      of[t][e] = (bf16)(((float)xr[t][e] - mean) * rstd * (float)gm[e] + (float)bt[e]);
  }

  // output tiles of 32 columns: o2^T tile = W^T rows x o1^T
  for (int nt = 0; nt < a.np / 32; ++nt) {
    const bf16* wrow = a.wt + (int64_t)(nt * 32 + l32) * LNL_K + 8 * g;
    f32x16 acc = {};
#pragma unroll
    for (int t = 0; t < NT; ++t) acc = M::mma(*(const bf16x8*)(wrow + 16 * t), of[t], acc);
    if (!mok) continue;
    // lane (row m, half g) holds columns nt 32 + 8 j + 4 g + 0..3
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = nt * 32 + 8 * j + 4 * g;
      if (col >= a.ncols) break;
      int i = 0;
#pragma unroll
      for (int u = 1; u < LNL_MAX_OUT; ++u) i += (u < a.n_out && col >= a.start[u]) ? 1 : 0;
      const int w = a.start[i + 1] - a.start[i];
      store4(a.out[i] + m * w + (col - a.start[i]),
             f32x4{acc[4 * j], acc[4 * j + 1], acc[4 * j + 2], acc[4 * j + 3]});
    }
  }
}

hipError_t launch_lnl_fwd(const LnlArgs& a, bf16* wt, const bf16* w, hipStream_t s) {
  {
    KernelTimer t(K_LNL_PREP, s);
    const int64_t nw = (int64_t)a.np * LNL_K;
    hipLaunchKernelGGL(lnl_wt_kernel, dim3((unsigned)((nw + 255) / 256)), dim3(256), 0, s, w,
                       a.ncols, a.np, wt);
  }
  LnlArgs b = a;
  b.wt = wt;
  {
    KernelTimer t(K_LNL_FWD, s);
    hipLaunchKernelGGL(lnl_fwd_kernel, dim3((unsigned)((a.m + 127) / 128)), dim3(256), 0, s, b);
  }
  return hipGetLastError();
}

}  // namespace triattn
