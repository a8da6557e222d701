// Wavefront helpers shared by the device sources.
#pragma once

#include "tfg_internal.h"

namespace tfg {

// A value the compiler cannot prove wave-uniform, made scalar.
__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

}  // namespace tfg
