// wf_decode_noalloc: the decode of wf_decode for callers that cannot allocate
// device memory.  The per-call working memory of a decode -- the hoisted
// hyperprior half of layer 1, the per-step activations, the old-tap context
// parts, the bf16 pair copy of y_hat and the call's pointer block -- is taken
// from one static device array of this file instead of the plan's workspace.
// The kernels are the per-step kernels of the stream driver, unchanged.
#include <algorithm>
#include <mutex>

#include "wf_device.h"

namespace wf {

// Each device that loads this library holds its own copy of the array until
// the process ends.  In host code `scratch` names a host-side stand-in, not
// device memory: only the address obtained with hipGetSymbolAddress (one per
// device, kept in scratch_dev) is ever passed to a kernel.
constexpr size_t kScratchBytes = 32u << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kScratchMaxDevices = 64;
static std::mutex scratch_mu;
static void* scratch_dev[kScratchMaxDevices];

// The device address of the current device's array (looked up once per device).
static int scratch_base(unsigned char** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(WF_E_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
    if (dev < 0 || dev >= kScratchMaxDevices) return fail(WF_E_UNSUPPORTED, "device index out of range");
    std::lock_guard<std::mutex> g(scratch_mu);
    if (!scratch_dev[dev]) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr)
            return fail(WF_E_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
        scratch_dev[dev] = ptr;
    }
    *out = static_cast<unsigned char*>(scratch_dev[dev]);
    return WF_OK;
}

// Carve the working memory of plan p out of [base, base + kScratchBytes):
// sub-arrays in order, each 256-byte aligned.  With base == nullptr only the
// size is computed.  Returns the bytes needed.
static size_t carve(const Plan& p, unsigned char* base, StepArgs& a, CallPtrs** cp) {
    const bool bf = p.precision == WF_BF16;
    const size_t MR = (size_t)p.max_rows, M = (size_t)p.M;
    const size_t nlat = (size_t)p.B * p.H * p.W;
    const int nparts = std::max(kCtxPartsMax, p.group > 1 ? a.gparts : 0);
    size_t off = 0;
    auto take = [&](size_t bytes) -> unsigned char* {
        unsigned char* q = base ? base + off : nullptr;
        off += (bytes + 255) / 256 * 256;
        return q;
    };
    *cp = reinterpret_cast<CallPtrs*>(take(sizeof(CallPtrs)));
    a.p1 = reinterpret_cast<float*>(take(nlat * p.Np1 * sizeof(float)));
    // h1, h2: four bytes per value (fp32, or a bf16 hi/lo pair)
    a.h1 = take(MR * p.Np1 * 4);
    a.h2 = take(MR * p.Np2 * 4);
    a.h2b = a.h2;
    a.ctxo = reinterpret_cast<float*>(take((size_t)2 * nparts * MR * 2 * M * sizeof(float)));
    a.ybf = bf ? reinterpret_cast<uint16_t*>(take(nlat * 2 * M * sizeof(uint16_t))) : nullptr;
    return off;
}

}  // namespace wf

using namespace wf;

extern "C" int wf_decode_noalloc(wf_plan_t plan, const float* psi, const int32_t* sym, const wf_out* out,
                                 hipStream_t stream) {
    if (!plan || !psi || !sym) return fail(WF_E_INVALID, "plan, psi or sym is NULL");
    if (!out || !out->y_hat || !out->mean || !out->scale || !out->idx)
        return fail(WF_E_INVALID, "y_hat, mean, scale and idx outputs are required");
    Plan* p = reinterpret_cast<Plan*>(plan);
    if (p->K == 3 && (!out->weight || !out->comp_mean))
        return fail(WF_E_INVALID, "weight and comp_mean outputs are required for K = 3");
    StepArgs a = p->args;
    // the stream driver's launch sequence and its number of old-tap context parts
    a.ctx_parts = p->precision == WF_BF16 ? kCtxPartsBf16 : kCtxPartsF32;
    CallPtrs* cp = nullptr;
    const size_t need = carve(*p, nullptr, a, &cp);
    if (need > kScratchBytes)
        return fail(WF_E_UNSUPPORTED, "the decode needs " + std::to_string(need) + " bytes of working memory; "
                                      "wf_decode_noalloc holds " + std::to_string(kScratchBytes));
    unsigned char* base = nullptr;
    int rc = scratch_base(&base);
    if (rc != WF_OK) return rc;
    carve(*p, base, a, &cp);
    a.cp = cp;
    CallPtrs c{};
    c.psi = psi; c.sym = sym; c.encode = 0;
    c.y_hat = out->y_hat; c.mean = out->mean; c.scale = out->scale; c.idx = out->idx;
    c.weight = out->weight; c.cmean = out->comp_mean;
    c.err = p->d_err;
    if ((rc = enqueue_set_call_at(cp, c, stream)) != WF_OK) return rc;
    return enqueue_steps_with(*p, a, stream);
}
