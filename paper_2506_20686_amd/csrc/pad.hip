// Head-dimension padding for d = 16: the d = 32 kernels run on tensors
// whose channels 16..31 are zero.  Zero channels add exact zeros to every
// logit and to no output channel that is kept, so the results for channels
// 0..15 are those of a d = 16 computation.
#include "kernels.h"
#include "timing.h"

namespace triattn {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// dst row r (2 cpr 16-byte chunks) = src row r (cpr chunks), then zeros.
__global__ __launch_bounds__(256) void pad_rows_kernel(const u32x4* src, u32x4* dst,
                                                       int64_t rows, int cpr) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= rows * 2 * cpr) return;
  const int64_t r = idx / (2 * cpr);
  const int c = (int)(idx % (2 * cpr));
  dst[idx] = c < cpr ? src[r * cpr + c] : u32x4{0u, 0u, 0u, 0u};
}

// dst row r (cpr chunks) = the first half of src row r (2 cpr chunks).
__global__ __launch_bounds__(256) void unpad_rows_kernel(const u32x4* src, u32x4* dst,
                                                         int64_t rows, int cpr) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= rows * cpr) return;
  const int64_t r = idx / cpr;
  const int c = (int)(idx % cpr);
  dst[idx] = src[r * 2 * cpr + c];
}

}  // namespace

hipError_t launch_pad16(const void* src, void* dst, int64_t rows, int elem_bytes,
                        hipStream_t s) {
  const int cpr = 16 * elem_bytes / 16;  // 16-byte chunks per unpadded row
  const int64_t n = rows * 2 * cpr;
  KernelTimer t(K_PAD, s);
  hipLaunchKernelGGL(pad_rows_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                     (const u32x4*)src, (u32x4*)dst, rows, cpr);
  return hipGetLastError();
}

hipError_t launch_unpad16(const void* src, void* dst, int64_t rows, int elem_bytes,
                          hipStream_t s) {
  const int cpr = 16 * elem_bytes / 16;
  const int64_t n = rows * cpr;
  KernelTimer t(K_PAD, s);
  hipLaunchKernelGGL(unpad_rows_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                     (const u32x4*)src, (u32x4*)dst, rows, cpr);
  return hipGetLastError();
}

}  // namespace triattn
