// noalloc.hip -- rgat_forward_noalloc: the RGAT forward with its workspace in
// a static device array instead of a caller buffer, for callers that cannot
// allocate device memory (code under HIP graph capture, serving loops,
// harnesses that forbid allocation).
//
// `scratch` below is a file-scope device array of kScratchBytes.  Every GPU
// the library runs on holds its own copy at its own address until the
// process ends.  Host code never uses the array's name as an address (on the
// host it is only a stand-in symbol): the device address is looked up once
// per device with hipGetSymbolAddress, with that device current, and only
// that address is passed on.  Calls that overlap on one GPU share the array
// and race; the caller serialises them (one stream, or events).  The layer
// writes every workspace entry before reading it, so the array needs no
// clearing between calls.
#include <mutex>
#include <string>

#include "rgnn_internal.h"

namespace rgnn {
namespace {

constexpr size_t kScratchBytes = size_t(64) << 20;   // 64 MiB per device
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];   // device address of `scratch` per device, once looked up

// Device address of `scratch` on the current device `dev`.
rgnn_status scratch_address(int dev, void **ptr)
{
    if (dev < 0 || dev >= kMaxDevices)
        return fail(RGNN_EUNSUPPORTED, "device id " + std::to_string(dev) + " beyond the scratch table");
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!p) return fail(RGNN_EDEVICE, "hipGetSymbolAddress(scratch) returned NULL");
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return RGNN_OK;
}

}  // namespace
}  // namespace rgnn

using namespace rgnn;

extern "C" rgnn_status rgat_forward_noalloc(const rgnn_graph_t *g, const float *h, const float *W,
                                            const float *w_src, const float *w_dst, int32_t d_in,
                                            int32_t d_out, int32_t heads, float neg_slope,
                                            int32_t softmax_scope, int32_t plan, float *out, float *saved,
                                            void *stream)
{
    if (!g) return fail(RGNN_EINVAL, "graph is NULL");
    // the workspace rgat_forward needs for these arguments (the per-(dst, rel)
    // softmax runs the aggregate-first plan)
    const int32_t ws_plan = softmax_scope == RGNN_SOFTMAX_PER_DST_REL ? (int32_t)RGNN_PLAN_AGGREGATE_FIRST : plan;
    size_t need = 0;
    rgnn_status st = rgnn_workspace_size(g, RGNN_LAYER_RGAT, d_in, d_out, heads, ws_plan, &need);
    if (st != RGNN_OK) return st;
    if (need > kScratchBytes)
        return fail(RGNN_ERANGE, "rgat_forward_noalloc: this graph and width need " + std::to_string(need) +
                                     " bytes of workspace; the static scratch holds " +
                                     std::to_string(kScratchBytes) + " bytes (use rgat_forward)");
    int dev = -1;
    const hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    void *ws = nullptr;
    if ((st = scratch_address(dev, &ws)) != RGNN_OK) return st;
    return rgat_forward(g, h, W, w_src, w_dst, d_in, d_out, heads, neg_slope, softmax_scope, plan, out, saved, ws,
                        kScratchBytes, stream);
}
