// Triangle-attention forward (MegaFold Section IV-A, "EvoFlash-3D" forward):
// per (row, head, block of queries) stream the key tiles of the row, keep a
// running max and sum (online softmax), rescale and accumulate the output,
// and save the log-sum-exp.  Also the per-call preparation kernels.
//
// Differences from the paper's Triton kernel, for gfx950:
//  - one workgroup = 4 waves = 128 queries of one (row, head); the K and V
//    tiles of the row are staged once in LDS and shared by the 4 waves;
//  - logits are formed transposed (S^T = K Q^T) so that each lane owns one
//    query: the running max/sum are per-lane scalars and the output
//    accumulator O^T = V^T P^T is rescaled with one multiply per register;
//  - the bias (pre-divided by the scale, laid out query-major) is the
//    initial MFMA accumulator, so adding it costs no vector instruction, and
//    the softmax runs in base 2 with scale * log2(e) folded into one FMA;
//  - the sigmoid gate is applied in the epilogue;
//  - key tiles that are fully masked for the row are skipped.
#include "kernels.h"
#include "stage.h"
#include "timing.h"

namespace triattn {

// ---- preparation ------------------------------------------------------------------

// bt[h][x][y] = bias(query x, key y, h) / scale and btT[h][x][y] =
// bias(query y, key x, h) / scale over the zero-padded np x np map.  The
// starting node reads bias[q][k][h], the ending node bias[k][q][h].
template <typename T>
__global__ __launch_bounds__(256) void prep_bias_kernel(Geom G, int node, const T* bias,
                                                        float* bt, float* btT) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t np = G.np, total = (int64_t)G.H * np * np;
  if (idx >= total) return;
  const int y = (int)(idx % np), x = (int)((idx / np) % np), h = (int)(idx / (np * np));
  const int n = G.n;
  auto at = [&](int qi, int ki) -> int64_t {
    return node == 0 ? ((int64_t)qi * n + ki) * G.H + h : ((int64_t)ki * n + qi) * G.H + h;
  };
  const bool in = x < n && y < n;
  bt[idx] = in ? (float)bias[at(x, y)] / G.scale : 0.f;
  if (btT) btT[idx] = in ? (float)bias[at(y, x)] / G.scale : 0.f;
}

// kbits[row][t]: bit e set iff key 32 t + e < n and mask(row, key) != 0.
// The starting node reads mask[row][key], the ending node mask[key][row].
__global__ __launch_bounds__(256) void prep_kbits_kernel(Geom G, int node, const uint8_t* mask,
                                                         uint32_t* kbits) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)G.n * G.nkt) return;
  const int row = (int)(idx / G.nkt), t = (int)(idx % G.nkt), n = G.n;
  uint32_t bits = 0;
  for (int e = 0; e < 32; ++e) {
    const int key = 32 * t + e;
    if (key >= n) break;
    const bool ok = mask == nullptr ||
                    mask[node == 0 ? (int64_t)row * n + key : (int64_t)key * n + row] != 0;
    bits |= (ok ? 1u : 0u) << e;
  }
  kbits[idx] = bits;
}

template <typename T>
hipError_t launch_prep(const Geom& g, int node, const T* bias, const uint8_t* mask, const Prep& p,
                       hipStream_t s) {
  const int64_t nb = ((int64_t)g.H * g.np * g.np + 255) / 256;
  {
    KernelTimer t(K_PREP_BIAS, s);
    hipLaunchKernelGGL(prep_bias_kernel<T>, dim3((unsigned)nb), dim3(256), 0, s, g, node, bias,
                       p.bt, p.btT);
  }
  const int64_t nk = ((int64_t)g.n * g.nkt + 255) / 256;
  {
    KernelTimer t(K_PREP_KBITS, s);
    hipLaunchKernelGGL(prep_kbits_kernel, dim3((unsigned)nk), dim3(256), 0, s, g, node, mask,
                       p.kbits);
  }
  return hipGetLastError();
}

// ---- forward ----------------------------------------------------------------------

constexpr int FWD_WAVES = 4;
constexpr int FWD_QBLK = FWD_WAVES * TILE;  // queries per workgroup

template <typename T>
struct FwdArgs {
  Geom g;
  const float* bt;
  const uint32_t* kbits;
  const T *q, *k, *v, *gate;
  T* out;
  float* lse;
  int nqb;  // query blocks per row
};

template <typename T>
__global__ __launch_bounds__(256) void fwd_kernel(FwdArgs<T> a) {
  using M = Mma<T>;
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int qb = w % a.nqb, rh = w / a.nqb;
  const int r = rh % G.n, h = rh / G.n;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int q0 = qb * FWD_QBLK + wave * TILE;  // first query of this wave
  const bool active = q0 < G.n;
  const int q = q0 + l32;
  const bool qok = q < G.n;

  __shared__ __align__(16) T ks[TILE * LDS_ROW];      // K tile  [key][channel]
  __shared__ __align__(16) T vt[HEAD_DIM * LDS_ROW];  // V^T tile [channel][key]

  const int64_t rowbase = (int64_t)r * G.sRow + (int64_t)h * HEAD_DIM;
  typename M::frag qf[M::KCH];
  if (qok)
    row_frags(a.q + rowbase + (int64_t)q * G.sPos, g, qf);
  else
    zero_frags<T>(qf);

  const float c1 = G.scale * LOG2E;
  float m = neg_inf(), lsum = 0.f;
  f32x16 o = {};
  const uint32_t* kb = a.kbits + (int64_t)r * G.nkt;
  const float* bq = a.bt + ((int64_t)h * G.np + (active ? q : 0)) * G.np + 4 * g;

  for (int kt = 0; kt < G.nkt; ++kt) {
    const uint32_t bits = kb[kt];
    if (bits == 0u) continue;  // no valid key in this tile (same for every wave)
    __syncthreads();
    if (tid < 128)
      stage_tile<true, false>(a.k + rowbase, G.sPos, kt * TILE, bits, tid, ks, (T*)nullptr);
    else
      stage_tile<false, true>(a.v + rowbase, G.sPos, kt * TILE, bits, tid - 128, (T*)nullptr, vt);
    __syncthreads();
    if (!active) continue;

    // s^T = bias + K Q^T for this lane's query and the tile's 32 keys
    f32x16 s;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const f32x4 x = *(const f32x4*)(bq + kt * TILE + 8 * j);
#pragma unroll
      for (int e = 0; e < 4; ++e) s[4 * j + e] = x[e];
    }
    typename M::frag kf[M::KCH];
    row_frags(ks + l32 * LDS_ROW, g, kf);
#pragma unroll
    for (int t = 0; t < M::KCH; ++t) s = M::mma(kf[t], qf[t], s);
    if (bits != 0xffffffffu) {
#pragma unroll
      for (int v = 0; v < 16; ++v)
        if (!((bits >> acc_row(v, g)) & 1u)) s[v] = neg_inf();
    }

    // online softmax in base 2: logit2 = s * scale * log2(e)
    float mx = s[0];
#pragma unroll
    for (int v = 1; v < 16; ++v) mx = fmaxf(mx, s[v]);
    mx = wave_xor32_max(mx);
    const float mnew = fmaxf(m, mx * c1);
    const float mu = mnew == neg_inf() ? 0.f : mnew;
    const float alpha = __builtin_amdgcn_exp2f(m - mu);
    float ps = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      s[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], c1, -mu));
      ps += s[v];
    }
    lsum = lsum * alpha + ps;
#pragma unroll
    for (int v = 0; v < 16; ++v) o[v] *= alpha;
    m = mnew;

    // O^T += V^T P^T
    typename M::frag pf[M::PCH], vf[M::PCH];
    acc_frags(s, pf);
    quad_frags(vt + l32 * LDS_ROW, g, vf);
#pragma unroll
    for (int t = 0; t < M::PCH; ++t) o = M::mma(vf[t], pf[t], o);
  }
  if (!active) return;

  // epilogue: normalise, gate, store; lse = ln(sum exp) = (m + log2 l) ln 2
  const float lt = wave_xor32_sum(lsum);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  if (!qok) return;
  const int64_t base = rowbase + (int64_t)q * G.sPos;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int c0 = 8 * j + 4 * g;
    const f32x4 gv = load4(a.gate + base + c0);
    f32x4 ov;
#pragma unroll
    for (int e = 0; e < 4; ++e) ov[e] = o[4 * j + e] * inv / (1.f + __expf(-gv[e]));
    store4(a.out + base + c0, ov);
  }
  if (g == 0)
    a.lse[(int64_t)r * G.lRow + (int64_t)q * G.lPos + h] =
        lt > 0.f ? (m + log2f(lt)) * LN2 : neg_inf();
}

template <typename T>
hipError_t launch_fwd(const Geom& g, const Prep& p, const T* q, const T* k, const T* v,
                      const T* gate, T* out, float* lse, hipStream_t s) {
  FwdArgs<T> a{g, p.bt, p.kbits, q, k, v, gate, out, lse, (g.n + FWD_QBLK - 1) / FWD_QBLK};
  const int64_t nwg = (int64_t)a.nqb * g.n * g.H;
  {
    KernelTimer t(K_FWD, s);
    hipLaunchKernelGGL(fwd_kernel<T>, dim3((unsigned)nwg), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

template hipError_t launch_prep<bf16>(const Geom&, int, const bf16*, const uint8_t*, const Prep&,
                                      hipStream_t);
template hipError_t launch_prep<float>(const Geom&, int, const float*, const uint8_t*,
                                       const Prep&, hipStream_t);
template hipError_t launch_fwd<bf16>(const Geom&, const Prep&, const bf16*, const bf16*,
                                     const bf16*, const bf16*, bf16*, float*, hipStream_t);
template hipError_t launch_fwd<float>(const Geom&, const Prep&, const float*, const float*,
                                      const float*, const float*, float*, float*, hipStream_t);

}  // namespace triattn
