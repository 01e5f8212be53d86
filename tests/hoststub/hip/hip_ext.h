// Stand-in for the AMD extensions of the HIP runtime used by libgemel's
// host sources (kernel launches that time the kernel with two events).
#pragma once
#include "hip_runtime.h"

extern "C" hipError_t hipExtLaunchKernel(const void *f, dim3 g, dim3 b, void **args, size_t shm, hipStream_t s,
                                         hipEvent_t start, hipEvent_t stop, int flags);
