// Host-only stand-in (see hip_runtime.h): the extended launch API is not used by the
// runtime itself, only by the kernels' sources, which the stub backend replaces.
#pragma once
#include <hip/hip_runtime.h>
