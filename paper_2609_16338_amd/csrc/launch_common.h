// Host-side helpers shared by the GEMV launchers.
#pragma once

#include <hip/hip_runtime.h>

#include "../../include/bitcos.h"

// Status of the launch just enqueued on this thread.
inline int bitcos_launch_status() {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? BITCOS_OK : BITCOS_E_HIP;
}
