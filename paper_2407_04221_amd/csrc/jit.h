// Run-time compilation of the kernels generated from a rule set (lane16).
#pragma once

#include <hip/hip_runtime.h>

#include <string>

namespace av {

// Compiles `source` with hipRTC for gfx950 and loads `kernel` from it on the current device.
// An identical earlier build on the same device is reused (modules stay loaded for the
// process).  On a compile failure returns hipErrorInvalidKernelFile and the compiler log in
// *log.
hipError_t jit_kernel(const std::string &source, const char *file_name, const char *kernel,
                      hipFunction_t *fn, std::string *log);

}  // namespace av
