// Persistent driver: one cooperative launch runs every wavefront step; the
// phases of a step are separated by a device-wide barrier instead of
// kernel boundaries.  Each workgroup loops over the jobs of a phase with a
// stride of the grid size (a multiple of 8, so a job's XCD placement is the
// same as in the per-step kernels), and all data that crosses workgroups
// inside the launch (h1, h2, y_hat, old-tap context) moves through agent-coherent
// (sc1) buffer accesses.
#include "wf_device.h"

namespace wf {

// Device-wide barrier, a three-level arrival tree and a release word per
// XCD class.  Workgroup g counts into group counter q = g % 64 (at most
// ceil(G / 64) arrivals per address); the last arrival of a group counts
// into class counter q % 8, the last of a class into the top counter, and
// the last arrival there publishes the round in eight release words, one per
// class g % 8, which that class's workgroups poll (at most G / 8 pollers per
// address).  Counters only grow: a round k completes when every level has
// counted k times its arrivals.  A wait longer than `budget` wall-clock
// ticks records WF_E_TIMEOUT in *err; every workgroup that sees a recorded
// error leaves the kernel at its next barrier, so the grid always drains.
struct Trace {
    long long* stamps;   // optional: arrival/leave wall-clock ticks per barrier
    long long cap;
    unsigned stall;      // test hook: 1 makes every barrier wait unreachable
};

constexpr int kBarGroups = 64;                // first-level counters
constexpr int kBarSlot = 32;                  // words between counters (128 bytes)
// layout (in slots): groups [0, 64), classes [64, 72), top 72, release [73, 81)
static_assert((kBarGroups + 2 * kXcds + 1) * kBarSlot <= kBarrierWords, "barrier words");

__device__ __forceinline__ unsigned bar_count(unsigned G, unsigned q, unsigned stride) {
    return q < G ? (G - q + stride - 1) / stride : 0u;   // members of residue class q modulo stride
}

__device__ __forceinline__ bool grid_barrier(unsigned* ctr, unsigned k, int* err, long long budget,
                                             int* bail, const Trace& tr) {
    __builtin_amdgcn_s_waitcnt(0);  // this wave's coherent stores have landed
    __syncthreads();
    if (threadIdx.x == 0) {
        const long long slot = (long long)(k - 1) * (gridDim.x + 1);
        if (tr.stamps && slot + gridDim.x < tr.cap) tr.stamps[slot + blockIdx.x] = wall_clock64();
        const unsigned G = gridDim.x;
        const unsigned q = blockIdx.x % kBarGroups, x = q % kXcds;
        const unsigned ngroups = G < (unsigned)kBarGroups ? G : (unsigned)kBarGroups;
        const unsigned nclass = ngroups < (unsigned)kXcds ? ngroups : (unsigned)kXcds;
        unsigned* rel = ctr + (kBarGroups + kXcds + 1) * kBarSlot;
        if (__hip_atomic_fetch_add(ctr + q * kBarSlot, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1 ==
                k * bar_count(G, q, kBarGroups) &&
            __hip_atomic_fetch_add(ctr + (kBarGroups + x) * kBarSlot, 1u, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT) + 1 == k * bar_count(ngroups, x, kXcds) &&
            __hip_atomic_fetch_add(ctr + (kBarGroups + kXcds) * kBarSlot, 1u, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT) + 1 == k * nclass) {
            for (int y = 0; y < kXcds; ++y)
                __hip_atomic_store(rel + y * kBarSlot, k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        int flag = 0;
        const long long t0 = wall_clock64();
        unsigned it = 0;
        const unsigned* mine = rel + (blockIdx.x % kXcds) * kBarSlot;
        while (__hip_atomic_load(mine, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < k + tr.stall) {
            if ((++it & 255u) == 0) {
                if (__hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) {
                    flag = 1;
                    break;
                }
                if (wall_clock64() - t0 > budget) {
                    __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    flag = 1;
                    break;
                }
            }
        }
        *bail = flag;
        if (tr.stamps && blockIdx.x == 0 && slot + gridDim.x < tr.cap) tr.stamps[slot + gridDim.x] = wall_clock64();
    }
    __syncthreads();
    return *bail == 0;
}

// Two workgroups per CU (one hides the other's load latency): at most 256
// registers per lane.
template <class P, int KC>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_persistent(StepArgs a, int T, unsigned* ctr, int* err,
                                                    long long budget, Trace tr) {
    __shared__ f4 red[kWaves * kMaxC][64];
    __shared__ L3Smem<KC> sm;
    __shared__ int bail;
    for (int l = threadIdx.x; l < a.L; l += blockDim.x) sm.tab[l] = a.table[l];
    __syncthreads();
    const int G = gridDim.x;
    unsigned k = 0;
    // pre-loop: the hyperprior half of layer 1 for every latent, and the
    // old-tap context of step 0 (no old tap of step 0 lies in the grid, but
    // the general form keeps the loop uniform)
    {
        const int nh = hoist_blocks<2>(a);
        for (int b = blockIdx.x; b < nh; b += G) hoist_job<P, true, 2, P::kBf16 ? 6 : 8>(a, b);
        const StepRows s0 = step_rows(a.H, a.W, a.B, a.lambda, 0);
        const int nc = ctxo_blocks<P>(a, s0);
        // the last part adds the others, so it runs after them
        const int split = (P::kParts - 1) * nc;
        for (int b = blockIdx.x; b < split; b += G) ctxo_job<P, true>(a, s0, b, nc, red);
        if (!grid_barrier(ctr, ++k, err, budget, &bail, tr)) return;
        for (int b = split + blockIdx.x; b < P::kParts * nc; b += G) ctxo_job<P, true>(a, s0, b, nc, red);
        if (!grid_barrier(ctr, ++k, err, budget, &bail, tr)) return;
    }
    for (int t = 0; t < T; ++t) {
        const StepRows s = step_rows(a.H, a.W, a.B, a.lambda, t);
        StepRows s1{t + 1, 0, 0, 0, 0};
        if (t + 1 < T) s1 = step_rows(a.H, a.W, a.B, a.lambda, t + 1);
        const StepWork w = step_work<P>(a, s, s1);
        for (int ph = P::kFirst; ph < kMaxPhases; ++ph) {
            const int nb = w.blocks(ph), j0 = w.first(ph);
            for (int b = blockIdx.x; b < nb + w.first(ph + 1) - j0; b += G) {
                if (b < nb)
                    phase_job<P, KC, true>(ph, a, s, b, red, sm);
                else
                    ctxo_job<P, true>(a, s1, j0 + b - nb, w.nc, red);
            }
            if (!grid_barrier(ctr, ++k, err, budget, &bail, tr)) return;
        }
    }
}

__global__ void k_zero_u32(unsigned* p, int n) {
    for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0u;
}

static const void* persistent_fn(const Plan& p) {
    if (p.precision == WF_BF16)
        return p.K == 1 ? (const void*)k_persistent<PBF16, 1> : (const void*)k_persistent<PBF16, 3>;
    return p.K == 1 ? (const void*)k_persistent<PF32, 1> : (const void*)k_persistent<PF32, 3>;
}

// Grid size of the persistent kernel: two workgroups per CU when they fit (one
// hides the other's memory latency), else one; a multiple of 8 (XCD placement).
int persistent_grid(Plan& p, int* grid) { return coop_grid(p, persistent_fn(p), grid); }

int coop_grid(Plan& p, const void* fn, int* grid) {
    int dev = 0, cus = 0, per_cu = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess)
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kThreads, 0);
    if (e != hipSuccess) return fail(WF_E_HIP, std::string("occupancy query: ") + hipGetErrorString(e));
    if (p.cu_limit > 0 && p.cu_limit < cus) cus = p.cu_limit;
    if (per_cu < 1 || cus < kXcds)
        return fail(WF_E_UNSUPPORTED, "cooperative kernel cannot be resident (fewer than 8 compute units)");
    *grid = cus * (per_cu >= 2 ? 2 : 1) / kXcds * kXcds;
    return WF_OK;
}

int enqueue_persistent(Plan& p, hipStream_t stream) {
    hipLaunchKernelGGL(k_zero_u32, dim3(1), dim3(256), 0, stream, p.d_bar, kBarrierWords);
    StepArgs a = p.args;
    int T = p.T;
    unsigned* ctr = p.d_bar;
    int* err = p.d_err;
    long long budget = p.spin_budget;
    Trace tr{p.stamps, p.stamps_cap, (unsigned)p.stall};
    void* args[] = {&a, &T, &ctr, &err, &budget, &tr};
    hipError_t e = hipLaunchCooperativeKernel(persistent_fn(p), dim3(p.grid), dim3(kThreads), args, 0, stream);
    if (e != hipSuccess) return fail(WF_E_HIP, std::string("cooperative launch: ") + hipGetErrorString(e));
    return WF_OK;
}

__global__ void k_empty(int* p) {
    if (p && threadIdx.x == 0 && blockIdx.x == 0 && p[0] == 12345) p[1] = 1;
}

// `rounds` empty device-wide barrier rounds over the whole grid.
__global__ __launch_bounds__(kThreads) void k_barrier_rounds(unsigned* ctr, int* err, long long budget, int rounds) {
    __shared__ int bail;
    const Trace tr{nullptr, 0, 0u};
    for (int r = 1; r <= rounds; ++r)
        if (!grid_barrier(ctr, (unsigned)r, err, budget, &bail, tr)) return;
}

int measure_floor(Plan& p, float* node_us, float* barrier_us) {
#define WF_FLOOR(call)                                                                      \
    do {                                                                                    \
        hipError_t e_ = (call);                                                             \
        if (e_ != hipSuccess) {                                                             \
            if (g) (void)hipGraphDestroy(g);                                                \
            if (ge) (void)hipGraphExecDestroy(ge);                                          \
            if (st) (void)hipStreamDestroy(st);                                             \
            if (e0) (void)hipEventDestroy(e0);                                              \
            if (e1) (void)hipEventDestroy(e1);                                              \
            return fail(WF_E_HIP, std::string(#call) + ": " + hipGetErrorString(e_));       \
        }                                                                                   \
    } while (0)
    hipStream_t st = nullptr;
    hipGraph_t g = nullptr;
    hipGraphExec_t ge = nullptr;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    const int nodes = 512, rounds = 1024;
    float ms = 0.0f;
    WF_FLOOR(hipStreamCreateWithFlags(&st, hipStreamNonBlocking));
    WF_FLOOR(hipEventCreate(&e0));
    WF_FLOOR(hipEventCreate(&e1));
    // (i) a chain of empty kernels replayed from a graph: per-node latency
    WF_FLOOR(hipStreamBeginCapture(st, hipStreamCaptureModeThreadLocal));
    for (int i = 0; i < nodes; ++i) hipLaunchKernelGGL(k_empty, dim3(1), dim3(64), 0, st, nullptr);
    WF_FLOOR(hipStreamEndCapture(st, &g));
    WF_FLOOR(hipGraphInstantiate(&ge, g, nullptr, nullptr, 0));
    WF_FLOOR(hipGraphLaunch(ge, st));
    WF_FLOOR(hipEventRecord(e0, st));
    WF_FLOOR(hipGraphLaunch(ge, st));
    WF_FLOOR(hipEventRecord(e1, st));
    WF_FLOOR(hipEventSynchronize(e1));
    WF_FLOOR(hipEventElapsedTime(&ms, e0, e1));
    *node_us = ms * 1e3f / nodes;
    // (ii) empty device-wide barrier rounds over the persistent grid
    *barrier_us = -1.0f;
    int grid = p.grid;
    if (grid == 0 && persistent_grid(p, &grid) != WF_OK) grid = 0;
    if (grid > 0) {
        unsigned* ctr = nullptr;
        WF_FLOOR(hipMalloc((void**)&ctr, kBarrierWords * sizeof(unsigned)));
        int* err = p.d_err;
        long long budget = p.spin_budget;
        int r = rounds;
        void* args[] = {&ctr, &err, &budget, &r};
        // one untimed launch first: the first cooperative launch of a process
        // pays one-time costs (code object, first touch) that no decode pays
        hipError_t e = hipSuccess;
        for (int pass = 0; pass < 2 && e == hipSuccess; ++pass) {
            e = hipMemsetAsync(ctr, 0, kBarrierWords * sizeof(unsigned), st);
            if (e == hipSuccess && pass == 1) e = hipEventRecord(e0, st);
            if (e == hipSuccess)
                e = hipLaunchCooperativeKernel((const void*)k_barrier_rounds, dim3(grid), dim3(kThreads), args, 0,
                                               st);
        }
        if (e == hipSuccess) e = hipEventRecord(e1, st);
        if (e == hipSuccess) e = hipEventSynchronize(e1);
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
        (void)hipFree(ctr);
        WF_FLOOR(e);
        *barrier_us = ms * 1e3f / rounds;
    }
    (void)hipGraphExecDestroy(ge);
    (void)hipGraphDestroy(g);
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    (void)hipStreamDestroy(st);
    return WF_OK;
#undef WF_FLOOR
}

}  // namespace wf
