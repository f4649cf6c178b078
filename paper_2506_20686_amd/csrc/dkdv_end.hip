// Triangle-attention dK, dV of the ending node (bf16): the kernel body of
// dkdv_dma.h compiled with LLVM's max-ilp scheduler at four waves per SIMD
// (two at 64 channels).  The starting node's kernels are in dkdv.hip.
#include "dkdv_dma.h"

namespace triattn {

template <int D>
__global__ __launch_bounds__(64 * KD_WAVES) __attribute__((amdgpu_waves_per_eu(KdL<D>::WPE, KdL<D>::WPE)))
void dkdv_dma_end_kernel(BwdArgs<bf16> a) {
  dkdv_dma_body<D>(a);
}

hipError_t launch_dkdv_dma_end(const BwdArgs<bf16>& a, hipStream_t s) {
  const Geom& g = a.g;
  const int64_t nwg = (int64_t)a.nblk * ((g.nr + KD_ROWS - 1) / KD_ROWS) * g.H;
  const dim3 grid((unsigned)nwg, 1, (unsigned)g.batch), block(64 * KD_WAVES);
  if (g.d == 64)
    hipLaunchKernelGGL(dkdv_dma_end_kernel<64>, grid, block, 0, s, a);
  else if (g.d == 16)
    hipLaunchKernelGGL(dkdv_dma_end_kernel<16>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(dkdv_dma_end_kernel<32>, grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace triattn
