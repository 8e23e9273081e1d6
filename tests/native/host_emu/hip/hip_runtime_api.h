/* Host stand-in for <hip/hip_runtime_api.h>: the public header of the library includes it
 * for hipStream_t, which the emulated runtime defines. */
#pragma once
#include "hip_runtime.h"
