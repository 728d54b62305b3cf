// Per-step kernels (stream and graph drivers): one launch per phase of every
// wavefront step, after the pre-loop hoist of the hyperprior half of layer 1.
#include "wf_device.h"

namespace wf {

// Pre-loop: P1[lat][n] = b_hoist[n] + sum_k psi[lat][k] * W1[n][k]  (k < 2M)
__global__ __launch_bounds__(256) void k_hoist(int nlat, StepArgs a) {
    __shared__ f4 red[kWaves][64];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, kq = lane >> 4;
    const int ct = blockIdx.x, rt = blockIdx.y;
    const int r = rt * kTile + (lane & 15);
    const float* __restrict__ psi = a.cp->psi + (size_t)r * 2 * a.M + kq * 4;
    const int n = ct * kTile + (lane & 15);
    const float bias = a.b_hoist[n];
    auto la = [&](int kb) -> f4 {
        return r < nlat ? *reinterpret_cast<const f4*>(psi + kb * kTile) : zero4();
    };
    const float v = block_tile(red, a.wp_hoist, 2 * a.M / kTile, ct, la);
    const int ro = rt * kTile + kq * 4 + wave;
    if (ro < nlat) a.p1[(size_t)ro * a.Np1 + n] = v + bias;
}

// Phase A: layer 1 of step s (blocks [0, nb1)) and the push of step sp.
__global__ __launch_bounds__(256) void k_phase_a(StepRows s, StepRows sp, int nb1, StepArgs a) {
    __shared__ f4 red[kWaves][64];
    if ((int)blockIdx.x >= nb1)
        push_job<false>(a, sp, blockIdx.x - nb1);
    else
        l1_job<false>(a, s, blockIdx.x, red);
}

__global__ __launch_bounds__(256) void k_phase_b(StepRows s, StepArgs a) {
    __shared__ f4 red[kWaves][64];
    l2_job<false>(a, s, blockIdx.x, red);
}

template <int KC>
__global__ __launch_bounds__(256) void k_phase_c(StepRows s, StepArgs a) {
    __shared__ L3Smem<KC> sm;
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
    const int nlat = p.B * p.H * p.W;
    hipLaunchKernelGGL(k_hoist, dim3(p.Np1 / kTile, ntiles(nlat)), dim3(256), 0, stream, nlat, p.args);
    return WF_OK;
}

int enqueue_steps(Plan& p, hipStream_t stream) {
    const StepArgs& a = p.args;
    enqueue_hoist(p, stream);
    StepRows prev{0, 0, 0, 0};
    for (int t = 0; t < p.T; ++t) {
        const StepRows s = step_rows(p.H, p.W, p.B, p.lambda, t);
        const int nb1 = phase_a_l1_blocks(a, s);
        const int nbp = t >= 1 ? phase_a_push_blocks(a, prev, p.T) : 0;
        hipLaunchKernelGGL(k_phase_a, dim3(nb1 + nbp), dim3(256), 0, stream, s, prev, nb1, a);
        hipLaunchKernelGGL(k_phase_b, dim3(phase_b_blocks(a, s)), dim3(256), 0, stream, s, a);
        if (p.K == 1)
            hipLaunchKernelGGL(k_phase_c<1>, dim3(phase_c_blocks(a, s)), dim3(256), 0, stream, s, a);
        else
            hipLaunchKernelGGL(k_phase_c<3>, dim3(phase_c_blocks(a, s)), dim3(256), 0, stream, s, a);
        prev = s;
    }
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(WF_E_HIP, std::string("kernel launch: ") + hipGetErrorString(err));
    return WF_OK;
}

}  // namespace wf
