// hipRTC compilation and a per-process cache of the loaded kernels (see jit.h).
#include "jit.h"

#include <hip/hiprtc.h>

#include <map>
#include <mutex>
#include <vector>

namespace av {
namespace {
std::mutex g_mu;
std::map<std::string, hipFunction_t> g_cache;   // (device, kernel, source) -> kernel
}  // namespace

hipError_t jit_kernel(const std::string &source, const char *file_name, const char *kernel,
                      hipFunction_t *fn, std::string *log) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const std::string key = std::to_string(dev) + '\n' + kernel + '\n' + source;
    std::lock_guard<std::mutex> lock(g_mu);
    auto it = g_cache.find(key);
    if (it != g_cache.end()) {
        *fn = it->second;
        return hipSuccess;
    }
    hiprtcProgram prog;
    if (hiprtcCreateProgram(&prog, source.c_str(), file_name, 0, nullptr, nullptr) != HIPRTC_SUCCESS)
        return hipErrorInvalidValue;
    const char *opts[] = {"--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature",
                          "-Xclang", "-packed-fp32-ops"};
    const hiprtcResult rc = hiprtcCompileProgram(prog, int(sizeof opts / sizeof opts[0]), opts);
    if (rc != HIPRTC_SUCCESS) {
        size_t n = 0;
        hiprtcGetProgramLogSize(prog, &n);
        std::string text(n, '\0');
        if (n) hiprtcGetProgramLog(prog, &text[0]);
        if (log) *log = std::string(hiprtcGetErrorString(rc)) + ": " + text;
        hiprtcDestroyProgram(&prog);
        return hipErrorInvalidKernelFile;
    }
    size_t n = 0;
    hiprtcGetCodeSize(prog, &n);
    std::vector<char> code(n);
    hiprtcGetCode(prog, code.data());
    hiprtcDestroyProgram(&prog);
    hipModule_t mod;
    e = hipModuleLoadData(&mod, code.data());
    if (e != hipSuccess) return e;
    hipFunction_t f;
    e = hipModuleGetFunction(&f, mod, kernel);
    if (e != hipSuccess) return e;
    g_cache[key] = f;
    *fn = f;
    return hipSuccess;
}

}  // namespace av
