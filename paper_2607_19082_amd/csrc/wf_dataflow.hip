// Dataflow driver: one cooperative launch runs every job of every wavefront
// step, but without a device-wide barrier between phases.  Each job waits
// only for the jobs whose results it reads, or whose inputs it is about to
// overwrite, through counters that producers bump once their stores have
// landed; so the rows of a step move on to the next layer as soon as their
// own inputs are complete, and the off-critical-path work (the old-tap
// context of the next step) runs whenever a workgroup is free.
//
// Jobs (the same tile bodies as the other drivers, with agent-coherent
// exchange), per step t and 16-row tile rt:
//   CTX(t)   old-tap context k-parts of step t's latents, all but the last
//                                            reads y_hat of steps <= t-2
//   CTXL(t)  the last part, which adds the others in
//   A(t)     layer 1                         reads CTXL(t) and y_hat of step t-1
//   B(t)     layer 2                         reads A(t)
//   C0(t)    layer 3, mean columns: writes mean and y_hat
//   C1(t)    layer 3, scale columns: writes scale and index
// The plan lists them in a topological order (every dependency of a job
// comes earlier in the list), split into a critical list (A, B, C0, C1)
// and a context list (CTX, CTXL) per XCD class (the class of a job is its
// column tile mod 8, as in the other drivers).  Workgroups [0, ncrit) form the
// critical pool, the rest the context pool; workgroup g of class x = g mod 8
// runs entries k, k + n, k + 2n, ... of its pool's list x, where k is its
// index among its pool's workgroups of class x and n their number.  Every
// list is a subsequence of the global order, so a job only waits for jobs
// that come earlier, and the workgroup holding the earliest unfinished job
// has finished everything before it in its own list: that job can always run,
// and with every workgroup resident (cooperative launch) the grid never
// deadlocks.
//
// Ordering argument (why the waits below suffice; "C0(s) done" means every
// C0 job of step s has finished, which transitively means everything of
// every earlier step that C0 depends on):
//   - y_hat is written once per latent by C0.  A(t) reads the two newest taps,
//     from step t-1: it waits for C0(t-1).  CTX(t) reads taps of steps
//     <= t-2: it waits for C0(t-2).  C0(s) done implies C0(s-1) done
//     (C0(s) <- B(s) <- A(s) <- C0(s-1)).
//   - h1 (one buffer) is rewritten by A(t); its readers B(t-1) are done once
//     C0(t-1) is (C0(t-1) <- B(t-1)).
//   - h2 is double-buffered by step parity: B(t) rewrites what C0(t-2) and
//     C1(t-2) read; C0(t-2) is implied by B(t)'s wait for A(t), C1(t-2) is
//     waited for explicitly.
//   - The old-tap context is double-buffered by step parity: CTX(t) and
//     CTXL(t) rewrite what A(t-2) / CTXL(t-2) read, which are done once C0(t-2)
//     is.
//   - psi's hoisted part P1 is written by the pre-loop kernel before the launch.
#include "wf_device.h"

namespace wf {

// Counter slot of XCD class x in counter group g: slots are 64 bytes apart,
// so that the producers of one group (spread over 8 classes) do not contend
// for one address.
__device__ __forceinline__ unsigned* df_slot(unsigned* cnt, int g, int x) {
    return cnt + ((size_t)g * kXcds + x) * kDfSlotWords;
}

__host__ __device__ __forceinline__ int df_group(int nrt_max, int t, int kind, int rt) {
    return (t * kJobKinds + kind) * (nrt_max + 1) + rt;
}

// Jobs of one wait: counter group g must reach, in every class x, mult times
// the number of column tiles in [lo, hi) of class x.
struct DfWait {
    int g, lo, hi, mult;
};

// The plan constants the waits depend on.
struct DfGeom {
    int H, W, B, lambda, nrt_max, G, nct_ctx, nct_a, nct_b, npx;
};

// The waits of job (t, kind, rt): at most three, into w; returns their
// number.  (Host and device: the kernel takes its waits from here, and the
// race checks of the test suite read the same ones through wf_plan_deps.)
__host__ __device__ __forceinline__ int df_waits(const DfGeom& g, int t, int kind, int rt, DfWait (&w)[3]) {
    int nw = 0;
    auto step_total = [&](int tt, int k, int lo, int hi) {
        const int nrt = ntiles(step_rows(g.H, g.W, g.B, g.lambda, tt).nrows);
        w[nw++] = DfWait{df_group(g.nrt_max, tt, k, g.nrt_max), lo, hi, nrt};
    };
    switch (kind) {
        case JK_CTX:
            if (t >= 2) step_total(t - 2, JK_C0, 0, g.G);
            break;
        case JK_CTXL:
            w[nw++] = DfWait{df_group(g.nrt_max, t, JK_CTX, rt), 0, g.nct_ctx, g.npx};
            break;
        case JK_A:
            w[nw++] = DfWait{df_group(g.nrt_max, t, JK_CTXL, rt), 0, g.nct_ctx, 1};
            if (t >= 1) step_total(t - 1, JK_C0, 0, g.G);
            break;
        case JK_B:
            w[nw++] = DfWait{df_group(g.nrt_max, t, JK_A, rt), 0, g.nct_a, 1};
            if (t >= 2) step_total(t - 2, JK_C1, g.G, 2 * g.G);
            break;
        default:   // JK_C0, JK_C1
            w[nw++] = DfWait{df_group(g.nrt_max, t, JK_B, rt), 0, g.nct_b, 1};
            break;
    }
    return nw;
}
// The plan constants of the waits, for job columns of C column tiles.
__host__ __device__ __forceinline__ DfGeom df_geom(const StepArgs& a, int nrt_max, int C) {
    const int nct_n = 2 * a.M / kTile / C;
    return DfGeom{a.H, a.W, a.B, a.lambda, nrt_max, a.M / kTile, a.n_old > 0 ? nct_n : 0, a.Np1 / kTile / C,
                  a.Np2 / kTile / C, a.ctx_parts - 1};
}

// Wave 0 polls the (up to 3) waits; lanes 0..7 each watch one class.  A wait
// longer than `budget` wall-clock ticks, or an error recorded by another
// workgroup, makes the whole workgroup leave (returns false).
__device__ __forceinline__ bool df_wait_all(const DfArgs& d, const DfWait* w, int nw, int* err, long long budget,
                                            int* bail) {
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
        int flag = 0;
        for (int i = 0; i < nw && !flag; ++i) {
            const unsigned tgt =
                lane < kXcds ? (unsigned)(w[i].mult * cnt_range(w[i].lo, w[i].hi, lane) + d.stall) : 0u;
            const unsigned* p = df_slot(d.cnt, w[i].g, lane & (kXcds - 1));
            const long long t0 = wall_clock64();
            unsigned it = 0;
            while (true) {
                const unsigned v = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (__all(v >= tgt)) break;
                if ((++it & 63u) == 0) {
                    if (__hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) {
                        flag = 1;
                        break;
                    }
                    if (wall_clock64() - t0 > budget) {
                        if (lane == 0) __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        flag = 1;
                        break;
                    }
                }
                __builtin_amdgcn_s_sleep(1);
            }
        }
        if (lane == 0) *bail = flag;
    }
    __syncthreads();
    return *bail == 0;
}

template <class P, int KC>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_dataflow(
    StepArgs a, DfArgs d, int* err, long long budget) {
    __shared__ f4 red[kWaves * kMaxC][64];
    __shared__ L3Smem<KC> sm;
    __shared__ int bail;
    for (int l = threadIdx.x; l < a.L; l += blockDim.x) sm.tab[l] = a.table[l];
    __syncthreads();
    const int x = blockIdx.x % kXcds;
    const bool crit = (int)blockIdx.x < d.ncrit;
    const int lw = crit ? blockIdx.x / kXcds : (blockIdx.x - d.ncrit) / kXcds;
    const int nwg = crit ? d.ncrit / kXcds : (gridDim.x - d.ncrit) / kXcds;
    const int li = crit ? x : kXcds + x;
    const int2* list = d.jobs + d.off[li];
    const int n = d.off[li + 1] - d.off[li];
    const DfGeom geo = df_geom(a, d.nrt_max, P::kC);
    for (int p = lw; p < n; p += nwg) {
        const int2 c = list[p];
        const int t = c.x, kind = c.y & 15, part = (c.y >> 4) & 15, rt = (c.y >> 8) & 255, ct = c.y >> 16;
        const StepRows s = step_rows(a.H, a.W, a.B, a.lambda, t);
        DfWait w[3];
        const int nw = df_waits(geo, t, kind, rt, w);
        const long long e = 3LL * (d.off[li] + p);
        const bool rec = d.stamps && e + 2 < d.stamps_cap && threadIdx.x == 0;
        if (rec) d.stamps[e] = wall_clock64();
        if (!df_wait_all(d, w, nw, err, budget, &bail)) return;
        if (rec) d.stamps[e + 1] = wall_clock64();
        const Job jb{true, ct, rt};
        switch (kind) {
            case JK_CTX:
            case JK_CTXL:
                ctxo_tile<P, true>(a, s, kind == JK_CTX ? part : a.ctx_parts - 1, jb, red);
                break;
            case JK_A:
                if constexpr (P::kBf16) l1_fold_bf16_tile<true>(a, s, jb, red);
                else l1_fold_tile<true>(a, s, jb, red);
                break;
            case JK_B:
                l2_tile<P, true>(a, s, jb, red);
                break;
            default:
                l3_tile<P, KC, true>(a, s, jb, sm);
                break;
        }
        // every wave's coherent stores have landed before the count goes up
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (rec) d.stamps[e + 2] = wall_clock64();
        if (threadIdx.x == 0) {
            const int cx = ct % kXcds;
            __hip_atomic_fetch_add(df_slot(d.cnt, df_group(d.nrt_max, t, kind, rt), cx), 1u, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            if (kind == JK_C0 || kind == JK_C1)
                __hip_atomic_fetch_add(df_slot(d.cnt, df_group(d.nrt_max, t, kind, d.nrt_max), cx), 1u,
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// Zero n 16-byte words (grid-stride; a kernel rather than a memset node, so
// that the call can be captured into a graph by a caller).
__global__ void k_zero_u128(uint4* p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = uint4{0u, 0u, 0u, 0u};
}

const void* dataflow_fn(const Plan& p) {
    if (p.precision == WF_BF16)
        return p.K == 1 ? (const void*)k_dataflow<PBF16, 1> : (const void*)k_dataflow<PBF16, 3>;
    return p.K == 1 ? (const void*)k_dataflow<PF32, 1> : (const void*)k_dataflow<PF32, 3>;
}

// The job lists of a plan, in the topological order described above.
int build_dataflow(Plan& p, std::vector<int2>& lists, DfArgs& d, std::vector<int>* order) {
    const StepArgs& a = p.args;
    const bool bf = p.precision == WF_BF16;
    const int C = bf ? kColsBf16 : kColsF32;
    const int parts = a.ctx_parts;
    const int npx = parts - 1;
    const int nct_n = 2 * p.M / kTile / C;
    const int nct_ctx = a.n_old > 0 ? nct_n : 0;
    const int nct_a = p.Np1 / kTile / C, nct_b = p.Np2 / kTile / C, nct_c = 2 * (p.M / kTile);
    std::vector<std::vector<int2>> q(2 * kXcds);
    std::vector<std::vector<int>> qo(2 * kXcds);   // each entry's position in the global order
    int nglobal = 0;
    auto push = [&](int t, int kind, int part, int rt, int ct) {
        const int pool = kind == JK_CTX || kind == JK_CTXL ? 1 : 0;
        q[pool * kXcds + ct % kXcds].push_back(int2{t, kind | (part << 4) | (rt << 8) | (ct << 16)});
        qo[pool * kXcds + ct % kXcds].push_back(nglobal++);
    };
    auto nrt = [&](int t) { return ntiles(step_rows(p.H, p.W, p.B, p.lambda, t).nrows); };
    auto tiles = [&](int t, int kind, int part, int lo, int hi) {
        for (int rt = 0; rt < nrt(t); ++rt)
            for (int ct = lo; ct < hi; ++ct) push(t, kind, part, rt, ct);
    };
    auto ctx = [&](int t) {
        for (int part = 0; part < npx; ++part) tiles(t, JK_CTX, part, 0, nct_ctx);
    };
    ctx(0);
    tiles(0, JK_CTXL, 0, 0, nct_ctx);
    for (int t = 0; t < p.T; ++t) {
        tiles(t, JK_A, 0, 0, nct_a);
        if (t + 1 < p.T) ctx(t + 1);
        tiles(t, JK_B, 0, 0, nct_b);
        if (t + 1 < p.T) tiles(t + 1, JK_CTXL, 0, 0, nct_ctx);
        tiles(t, JK_C0, 0, 0, nct_c / 2);
        tiles(t, JK_C1, 0, nct_c / 2, nct_c);
    }
    lists.clear();
    if (order) order->clear();
    d.off[0] = 0;
    for (int x = 0; x < 2 * kXcds; ++x) {
        lists.insert(lists.end(), q[x].begin(), q[x].end());
        if (order) order->insert(order->end(), qo[x].begin(), qo[x].end());
        if (lists.size() > (size_t)INT32_MAX) return fail(WF_E_UNSUPPORTED, "too many dataflow jobs");
        d.off[x + 1] = (int)lists.size();
    }
    // fields must fit the job code: rt < 256, ct < 32768, part < 16
    if (p.max_rows / kTile > 255 || nct_a >= 32768 || nct_b >= 32768 || parts > 15)
        return fail(WF_E_UNSUPPORTED, "grid too large for the dataflow job code");
    d.nrt_max = p.max_rows / kTile;
    d.cnt_words = (size_t)p.T * kJobKinds * (d.nrt_max + 1) * kXcds * kDfSlotWords;
    return WF_OK;
}

int enqueue_dataflow(Plan& p, hipStream_t stream) {
    const size_t n16 = p.df.cnt_words / 4;
    hipLaunchKernelGGL(k_zero_u128, dim3(1024), dim3(256), 0, stream, reinterpret_cast<uint4*>(p.df.cnt), n16);
    int rc = enqueue_hoist(p, stream);
    if (rc != WF_OK) return rc;
    StepArgs a = p.args;
    DfArgs d = p.df;
    d.stamps = p.stamps;
    d.stamps_cap = p.stamps_cap;
    d.stall = p.stall;
    int* err = p.d_err;
    long long budget = p.spin_budget;
    void* args[] = {&a, &d, &err, &budget};
    hipError_t e = hipLaunchCooperativeKernel(dataflow_fn(p), dim3(p.grid), dim3(kThreads), args, 0, stream);
    if (e != hipSuccess) return fail(WF_E_HIP, std::string("cooperative launch: ") + hipGetErrorString(e));
    return WF_OK;
}

// The job lists and waits of a plan's geometry (host only, for the race
// checks): per job in list order, {t, kind, part, rt, ct, list, global
// position, number of waits, then three (group, lo, hi, mult)}; the counter
// groups it bumps are (t, kind, rt) and, for C0 and C1, (t, kind, nrt_max).
int dataflow_deps(Plan& p, std::vector<int32_t>& out) {
    std::vector<int2> lists;
    std::vector<int> order;
    DfArgs d{};
    int rc = build_dataflow(p, lists, d, &order);
    if (rc != WF_OK) return rc;
    const int C = p.precision == WF_BF16 ? kColsBf16 : kColsF32;
    const DfGeom geo = df_geom(p.args, d.nrt_max, C);
    out.clear();
    for (int li = 0; li < 2 * kXcds; ++li)
        for (int e = d.off[li]; e < d.off[li + 1]; ++e) {
            const int2 c = lists[e];
            const int t = c.x, kind = c.y & 15, part = (c.y >> 4) & 15, rt = (c.y >> 8) & 255, ct = c.y >> 16;
            DfWait w[3] = {};
            const int nw = df_waits(geo, t, kind, rt, w);
            const int32_t head[8] = {t, kind, part, rt, ct, li, order[e], nw};
            out.insert(out.end(), head, head + 8);
            for (int i = 0; i < 3; ++i) {
                const int32_t q[4] = {w[i].g, w[i].lo, w[i].hi, w[i].mult};
                out.insert(out.end(), q, q + 4);
            }
        }
    out.push_back(d.nrt_max);   // the last entry: nrt_max
    return WF_OK;
}

}  // namespace wf
