// Per-step kernels (stream and graph drivers): one launch per phase of every
// wavefront step, after the pre-loop hoist of the hyperprior half of layer 1.
#include "wf_device.h"

namespace wf {

// Pre-loop: the hyperprior half of layer 1 for every latent, several row
// tiles per wave (every weight operand feeds that many MFMA chains): fp32
// eight, two k-blocks a load batch (4K decode 11.60 against 11.71-11.75 ms
// with four and four; 11.64-11.78 with 8/1, 12/1, 12/2, 16/1, 6/4, 8/4, 4/8);
// bf16 four and three.
template <class P>
constexpr int kHoistRt = P::kBf16 ? 4 : 8;
template <class P>
__global__ __launch_bounds__(kThreads) void k_hoist(StepArgs a) {
    hoist_job<P, false, kHoistRt<P>, P::kBf16 ? 3 : 2>(a, blockIdx.x);
}

// Old-tap context jobs [j0, ...) of step s1 only (before the first step).
template <class P>
__global__ __launch_bounds__(kThreads) void k_ctxo(StepRows s1, int j0, int nc, StepArgs a) {
    __shared__ f4 red[kWaves * kMaxC][64];
    ctxo_job<P, false>(a, s1, j0 + blockIdx.x, nc, red);
}

// Grouped decode: the context jobs of group s (all parts), for masks of at
// most NT taps.
template <class P, int NT>
__global__ __launch_bounds__(kThreads) void k_gctx(StepRows s, int nc, StepArgs a) {
    __shared__ f4 red[kWaves * kMaxC][64];
    gctx_job<P, NT, false>(a, s, blockIdx.x, nc, red);
}

// Phase ph of step s (blocks [0, nb)), then old-tap context jobs [j0, ...)
// of step s1.  EC: the decode from rANS streams (its phase C job holds more
// registers, so it is a kernel of its own).
template <class P, int KC, bool EC = false>
__global__ __launch_bounds__(kThreads) void k_phase(int ph, StepRows s, StepRows s1, int nb, int j0, int nc,
                                                    StepArgs a) {
    __shared__ f4 red[kWaves * kMaxC][64];
    __shared__ L3Smem<KC> sm;
    if ((int)blockIdx.x >= nb) {
        ctxo_job<P, false>(a, s1, j0 + blockIdx.x - nb, nc, red);
        return;
    }
    if (ph == PH_C) {
        for (int l = threadIdx.x; l < a.L; l += blockDim.x) sm.tab[l] = a.table[l];
        __syncthreads();
    }
    phase_job<P, KC, false, EC>(ph, a, s, blockIdx.x, red, sm);
}

__global__ void k_set_call(CallPtrs* dst, CallPtrs v) {
    if (threadIdx.x == 0) *dst = v;
}

int enqueue_set_call(Plan& p, const CallPtrs& c, hipStream_t stream) {
    return enqueue_set_call_at(p.d_call, c, stream);
}

int enqueue_set_call_at(CallPtrs* dst, const CallPtrs& c, hipStream_t stream) {
    hipLaunchKernelGGL(k_set_call, dim3(1), dim3(64), 0, stream, dst, c);
    return WF_OK;
}

template <class P>
static void launch_hoist(const StepArgs& a, hipStream_t stream) {
    hipLaunchKernelGGL(k_hoist<P>, dim3(hoist_blocks<kHoistRt<P>>(a)), dim3(kThreads), 0, stream, a);
}

int enqueue_hoist(Plan& p, hipStream_t stream) {
    if (p.precision == WF_BF16)
        launch_hoist<PBF16>(p.args, stream);
    else
        launch_hoist<PF32>(p.args, stream);
    return WF_OK;
}

// Rows of step t, or an empty step past the end.
static StepRows rows_of(const Plan& p, int t) {
    if (t >= p.T) return StepRows{t, 0, 0, 0, 0};
    return step_rows(p.H, p.W, p.B, p.lambda, t);
}

// Grouped decode: per group, the context (with fill), then layers 1-3.
template <class P, int KC>
static void launch_groups(const Plan& p, const StepArgs& a, hipStream_t stream) {
    launch_hoist<P>(a, stream);
    const int ncx = 2 * a.M / kTile / P::kC;
    for (int g = 0; g < p.steps; ++g) {
        const StepRows s{g, 0, 0, p.g_n[g], p.g_r0[g]};
        const int nrt = ntiles(s.nrows);
        const int nc = xcd_blocks(ncx, nrt);
        if (p.ntaps <= kTaps5x5)
            hipLaunchKernelGGL((k_gctx<P, kTaps5x5>), dim3(nc * a.gparts), dim3(kThreads), 0, stream, s, nc, a);
        else
            hipLaunchKernelGGL((k_gctx<P, kMaxTaps>), dim3(nc * a.gparts), dim3(kThreads), 0, stream, s, nc, a);
        const int nb[3] = {xcd_blocks(a.Np1 / kTile / P::kC, nrt), phase_blocks<P>(a, s, PH_B),
                           phase_blocks<P>(a, s, PH_C)};
        const int ph[3] = {PH_GA, PH_B, PH_C};
        for (int k = 0; k < 3; ++k)
            hipLaunchKernelGGL((k_phase<P, KC>), dim3(nb[k]), dim3(kThreads), 0, stream, ph[k], s, s, nb[k], 0, 0, a);
    }
}

template <class P, int KC>
static void launch_steps(const Plan& p, StepArgs a, hipStream_t stream, bool ec) {
    a.ec = ec ? 1 : 0;
    if (p.group > 1) {
        launch_groups<P, KC>(p, a, stream);
        return;
    }
    launch_hoist<P>(a, stream);
    {
        const StepRows s0 = rows_of(p, 0);
        const int nc = ctxo_blocks<P>(a, s0);
        // the last part adds the others, so it runs after them
        const int split = (P::kParts - 1) * nc;
        if (nc > 0) {
            hipLaunchKernelGGL(k_ctxo<P>, dim3(split), dim3(kThreads), 0, stream, s0, 0, nc, a);
            if (split < P::kParts * nc)
                hipLaunchKernelGGL(k_ctxo<P>, dim3(P::kParts * nc - split), dim3(kThreads), 0, stream, s0, split, nc,
                                   a);
        }
    }
    for (int t = 0; t < p.T; ++t) {
        const StepRows s = rows_of(p, t), s1 = rows_of(p, t + 1);
        const StepWork w = step_work<P>(a, s, s1);
        for (int ph = P::kFirst; ph < kMaxPhases; ++ph) {
            const int n = w.nb[ph] + w.cut[ph + 1] - w.cut[ph];
            if (ec && ph == PH_C)
                hipLaunchKernelGGL((k_phase<P, KC, true>), dim3(n), dim3(kThreads), 0, stream, ph, s, s1, w.nb[ph],
                                   w.cut[ph], w.nc, a);
            else
                hipLaunchKernelGGL((k_phase<P, KC>), dim3(n), dim3(kThreads), 0, stream, ph, s, s1, w.nb[ph],
                                   w.cut[ph], w.nc, a);
        }
    }
}

int enqueue_steps(Plan& p, hipStream_t stream, bool ec) { return enqueue_steps_with(p, p.args, stream, ec); }

int enqueue_steps_with(const Plan& p, const StepArgs& a, hipStream_t stream, bool ec) {
    if (p.precision == WF_BF16) {
        if (p.K == 1) launch_steps<PBF16, 1>(p, a, stream, ec);
        else launch_steps<PBF16, 3>(p, a, stream, ec);
    } else {
        if (p.K == 1) launch_steps<PF32, 1>(p, a, stream, ec);
        else launch_steps<PF32, 3>(p, a, stream, ec);
    }
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(WF_E_HIP, std::string("kernel launch: ") + hipGetErrorString(err));
    return WF_OK;
}

}  // namespace wf
