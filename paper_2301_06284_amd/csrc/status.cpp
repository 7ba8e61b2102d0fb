// status.cpp -- the library's error state: the thread-local message behind
// rgnn_last_error() and the helpers that set it.  Host code only; the graph
// index builder and these helpers link without any kernel.
#include <string>

#include "rgnn_internal.h"

namespace rgnn {

namespace {
thread_local std::string g_err;
}

rgnn_status fail(rgnn_status st, const std::string &msg)
{
    g_err = msg;
    return st;
}

rgnn_status hip_fail(hipError_t e, const char *what)
{
    g_err = std::string(what) + ": " + hipGetErrorString(e);
    return RGNN_EDEVICE;
}

}  // namespace rgnn

extern "C" const char *rgnn_last_error(void) { return rgnn::g_err.c_str(); }
extern "C" const char *rgnn_version(void) { return "librgnn 0.2 (gfx950, fp32)"; }
