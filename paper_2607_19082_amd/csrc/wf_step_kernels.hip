// Per-step kernels (stream and graph drivers): one launch per phase of every
// wavefront step, after the pre-loop hoist of the hyperprior half of layer 1.
#include "wf_device.h"

namespace wf {

// Pre-loop: the hyperprior half of layer 1 for every latent.
__global__ __launch_bounds__(kThreads) void k_hoist(StepArgs a) {
    __shared__ f4 red[kWaves][64];
    hoist_job<false>(a, blockIdx.x, red);
}

// Phase A: layer 1 of step s (blocks [0, nb)), then old-tap context jobs
// [j0, ...) of step s1.
__global__ __launch_bounds__(kThreads) void k_phase_a(StepRows s, StepRows s1, int nb, int j0, int nc, StepArgs a) {
    __shared__ f4 red[kWaves][64];
    if ((int)blockIdx.x < nb)
        l1_job<false>(a, s, blockIdx.x, red);
    else
        ctxo_job<false>(a, s1, j0 + blockIdx.x - nb, nc, red);
}

// Old-tap context jobs of step s1 only (before the first step).
__global__ __launch_bounds__(kThreads) void k_ctxo(StepRows s1, int nc, StepArgs a) {
    __shared__ f4 red[kWaves][64];
    ctxo_job<false>(a, s1, blockIdx.x, nc, red);
}

// Phase B: layer 2 of step s, then old-tap context jobs.
__global__ __launch_bounds__(kThreads) void k_phase_b(StepRows s, StepRows s1, int nb, int j0, int nc, StepArgs a) {
    __shared__ f4 red[kWaves][64];
    if ((int)blockIdx.x < nb)
        l2_job<false>(a, s, blockIdx.x, red);
    else
        ctxo_job<false>(a, s1, j0 + blockIdx.x - nb, nc, red);
}

// Phase C: layer 3 and the epilogue of step s, then old-tap context jobs.
template <int KC>
__global__ __launch_bounds__(kThreads) void k_phase_c(StepRows s, StepRows s1, int nb, int j0, int nc, StepArgs a) {
    __shared__ L3Smem<KC> sm;
    __shared__ f4 red[kWaves][64];
    if ((int)blockIdx.x >= nb) {
        ctxo_job<false>(a, s1, j0 + blockIdx.x - nb, nc, red);
        return;
    }
    for (int l = threadIdx.x; l < a.L; l += blockDim.x) sm.tab[l] = a.table[l];
    __syncthreads();
    l3_job<KC, false>(a, s, blockIdx.x, sm);
}

__global__ void k_set_call(CallPtrs* dst, CallPtrs v) {
    if (threadIdx.x == 0) *dst = v;
}

int enqueue_set_call(Plan& p, const CallPtrs& c, hipStream_t stream) {
    hipLaunchKernelGGL(k_set_call, dim3(1), dim3(64), 0, stream, p.d_call, c);
    return WF_OK;
}

int enqueue_hoist(Plan& p, hipStream_t stream) {
    hipLaunchKernelGGL(k_hoist, dim3(hoist_blocks(p.args)), dim3(kThreads), 0, stream, p.args);
    return WF_OK;
}

// Rows of step t, or an empty step past the end.
static StepRows rows_of(const Plan& p, int t) {
    if (t >= p.T) return StepRows{t, 0, 0, 0};
    return step_rows(p.H, p.W, p.B, p.lambda, t);
}

int enqueue_steps(Plan& p, hipStream_t stream) {
    const StepArgs& a = p.args;
    enqueue_hoist(p, stream);
    {
        const StepRows s0 = rows_of(p, 0);
        const int nc = ctxo_blocks(a, s0);
        if (nc > 0) hipLaunchKernelGGL(k_ctxo, dim3(kCtxParts * nc), dim3(kThreads), 0, stream, s0, nc, a);
    }
    for (int t = 0; t < p.T; ++t) {
        const StepRows s = rows_of(p, t), s1 = rows_of(p, t + 1);
        const int nc = ctxo_blocks(a, s1);
        const int nb1 = l1_blocks(a, s), nb2 = l2_blocks(a, s), nb3 = l3_blocks(a, s);
        int ka, kb, kc, ko;
        job_costs(a, &ka, &kb, &kc, &ko);
        const CtxSplit cs = ctxo_split(nc, nb1, nb2, nb3, ka, kb, kc, ko);
        hipLaunchKernelGGL(k_phase_a, dim3(nb1 + cs.c1), dim3(kThreads), 0, stream, s, s1, nb1, 0, nc, a);
        hipLaunchKernelGGL(k_phase_b, dim3(nb2 + cs.c2 - cs.c1), dim3(kThreads), 0, stream, s, s1, nb2, cs.c1, nc, a);
        if (p.K == 1)
            hipLaunchKernelGGL(k_phase_c<1>, dim3(nb3 + cs.total - cs.c2), dim3(kThreads), 0, stream, s, s1, nb3, cs.c2,
                               nc, a);
        else
            hipLaunchKernelGGL(k_phase_c<3>, dim3(nb3 + cs.total - cs.c2), dim3(kThreads), 0, stream, s, s1, nb3, cs.c2,
                               nc, a);
    }
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(WF_E_HIP, std::string("kernel launch: ") + hipGetErrorString(err));
    return WF_OK;
}

}  // namespace wf
