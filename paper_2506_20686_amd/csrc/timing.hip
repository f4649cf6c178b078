// Opt-in per-kernel timing: when enabled, each kernel launch of the library
// is bracketed by two HIP events recorded on the launch's stream; reading
// the timings waits for those events and accumulates their elapsed times
// per kernel.  Off by default, in which case the brackets cost one branch.
#include <mutex>
#include <vector>

#include "common.h"
#include "timing.h"
#include "triattn.h"

namespace triattn {

namespace {

const char* const kNames[K_COUNT] = {"prep_bias",   "prep_kbits", "fwd",        "bwd_prep",
                                     "bwd_pad",     "dq",         "dkdv",       "db",
                                     "db_reduce",   "lnl_fwd",    "lnl_bwd_dx",
                                     "lnl_bwd_g",   "lnl_reduce", "lnl_finish",
                                     "trn_pack",    "trn_fwd",    "trn_bwd_dx",
                                     "trn_bwd_w",   "trn_reduce", "trn_finish",
                                     "pad16"};

struct Pending {
  int id;
  hipEvent_t a, b;
};

struct State {
  std::mutex mu;
  bool on = false;
  uint64_t mask = 0;  // kernels timed (bit per KernelId); 0: all
  std::vector<hipEvent_t> pool;  // created events not in use
  std::vector<Pending> pending;  // recorded, not yet read
  double ms[K_COUNT] = {};
  int64_t launches[K_COUNT] = {};
  int status = TRIATTN_OK;
};

State& st() {
  static State s;
  return s;
}

bool take(State& s, hipEvent_t* e) {
  if (!s.pool.empty()) {
    *e = s.pool.back();
    s.pool.pop_back();
    return true;
  }
  return hipEventCreate(e) == hipSuccess;
}

void drain(State& s) {
  for (const Pending& p : s.pending) {
    float ms = 0.f;
    if (hipEventSynchronize(p.b) != hipSuccess || hipEventElapsedTime(&ms, p.a, p.b) != hipSuccess)
      s.status = TRIATTN_ERR_HIP;
    s.ms[p.id] += ms;
    s.launches[p.id] += 1;
    s.pool.push_back(p.a);
    s.pool.push_back(p.b);
  }
  s.pending.clear();
}

}  // namespace

KernelTimer::KernelTimer(KernelId id, hipStream_t stream) : id_(id), stream_(stream) {
  State& s = st();
  if (!s.on || (s.mask != 0 && !((s.mask >> id) & 1u))) return;
  std::lock_guard<std::mutex> lock(s.mu);
  if (!take(s, &a_) || !take(s, &b_) || hipEventRecord(a_, stream_) != hipSuccess) {
    s.status = TRIATTN_ERR_HIP;
    return;
  }
  armed_ = true;
}

KernelTimer::~KernelTimer() {
  if (!armed_) return;
  State& s = st();
  std::lock_guard<std::mutex> lock(s.mu);
  if (hipEventRecord(b_, stream_) != hipSuccess) {
    s.status = TRIATTN_ERR_HIP;
    return;
  }
  s.pending.push_back(Pending{id_, a_, b_});
  if (s.pending.size() >= 4096) drain(s);
}

}  // namespace triattn

extern "C" {

int tri_attn_timing_enable(int on) {
  triattn::State& s = triattn::st();
  std::lock_guard<std::mutex> lock(s.mu);
  s.on = on != 0;
  return TRIATTN_OK;
}

int tri_attn_timing_select(uint64_t mask) {
  triattn::State& s = triattn::st();
  std::lock_guard<std::mutex> lock(s.mu);
  s.mask = mask;
  return TRIATTN_OK;
}

int tri_attn_timing_reset(void) {
  triattn::State& s = triattn::st();
  std::lock_guard<std::mutex> lock(s.mu);
  triattn::drain(s);
  for (int i = 0; i < triattn::K_COUNT; ++i) {
    s.ms[i] = 0.0;
    s.launches[i] = 0;
  }
  const int r = s.status;
  s.status = TRIATTN_OK;
  return r;
}

int tri_attn_timing_read(int index, const char** name, double* total_ms, int64_t* launches) {
  if (index < 0 || index >= triattn::K_COUNT || name == nullptr || total_ms == nullptr ||
      launches == nullptr)
    return TRIATTN_ERR_INVALID_ARG;
  triattn::State& s = triattn::st();
  std::lock_guard<std::mutex> lock(s.mu);
  triattn::drain(s);
  *name = triattn::kNames[index];
  *total_ms = s.ms[index];
  *launches = s.launches[index];
  return s.status;
}

}  // extern "C"

// ---- MFMA counter calibration -------------------------------------------------------
//
// A kernel whose only work is bf16 MFMA: every wave runs `iters` rounds of
// eight v_mfma_f32_32x32x16_bf16 over four independent accumulator chains
// (4 waves per block, one per SIMD).  Profiled beside the attention kernels it
// gives the reading of the MFMA-activity counters for a known amount of MFMA
// work at full occupancy of the matrix cores.
namespace triattn {
namespace {

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 4)))
void mfma_probe_kernel(float* out, int iters) {
  bf16x8 a, b;
  const float x = 1.f + 1e-3f * (float)threadIdx.x;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (bf16)(x + (float)i);
    b[i] = (bf16)(x - (float)i);
  }
  f32x16 acc[4] = {};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int k = 0; k < 8; ++k)
      acc[k & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[k & 3], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int v = 0; v < 16; ++v) s += acc[m][v];
  out[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

}  // namespace
}  // namespace triattn

extern "C" int tri_attn_mfma_probe(int64_t blocks, int64_t iters, float* out, void* stream) {
  if (blocks < 1 || blocks > (1 << 20) || iters < 1 || iters > (1 << 24) || out == nullptr)
    return TRIATTN_ERR_INVALID_ARG;
  hipLaunchKernelGGL(triattn::mfma_probe_kernel, dim3((unsigned)blocks), dim3(256), 0,
                     (hipStream_t)stream, out, (int)iters);
  return hipGetLastError() == hipSuccess ? TRIATTN_OK : TRIATTN_ERR_HIP;
}
