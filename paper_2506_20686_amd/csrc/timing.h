// Per-kernel timing brackets (see timing.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace triattn {

enum KernelId {
  K_PREP_BIAS,
  K_PREP_KBITS,
  K_FWD,
  K_BWD_PREP,
  K_BWD_PAD,
  K_DQ,
  K_DKDV,
  K_DB,
  K_DB_REDUCE,
  K_LNL_FWD,
  K_LNL_BWD_DX,
  K_LNL_BWD_G,
  K_LNL_REDUCE,
  K_LNL_FINISH,
  K_TRN_PACK,
  K_TRN_FWD,
  K_TRN_BWD_DX,
  K_TRN_BWD_W,
  K_TRN_REDUCE,
  K_TRN_FINISH,
  K_PAD,
  K_COUNT
};

// Records an event on `stream` now and another when it goes out of scope,
// if timing is enabled; otherwise does nothing.
class KernelTimer {
 public:
  KernelTimer(KernelId id, hipStream_t stream);
  ~KernelTimer();
  KernelTimer(const KernelTimer&) = delete;
  KernelTimer& operator=(const KernelTimer&) = delete;

 private:
  int id_;
  hipStream_t stream_;
  hipEvent_t a_{}, b_{};
  bool armed_ = false;
};

}  // namespace triattn
