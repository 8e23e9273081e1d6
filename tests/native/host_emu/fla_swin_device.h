// Host build of the fp32 attention kernels and the Cycle-scan kernels: they need only the
// internal header (the bf16 kernels' vector types and matrix-core builtins are not built here),
// and the Cycle-scan kernels the hardware exp2, here the C library's.
#pragma once
#include <cmath>

#include "fla_swin_internal.h"

#define __builtin_amdgcn_exp2f(x) std::exp2((float)(x))
