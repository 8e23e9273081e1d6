// Host build of the fp32 kernels: they need only the internal header (the bf16 kernels' vector
// types and matrix-core builtins are not built here).
#pragma once
#include "fla_swin_internal.h"
