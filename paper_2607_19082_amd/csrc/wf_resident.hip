// Resident driver: one cooperative launch of two workgroups per compute unit.
// Every workgroup keeps one slice of the weights in registers for the whole
// decode and plays one fixed role:
//   CTX(c, p)  old-tap context, column tile c of 2M, k-part p < P-1 of the
//              old taps
//   CTXL(c)    the same for the last part P-1, which also adds the other
//              parts' results (so layer 1 reads one context value)
//   A(c)       layer 1 over [new taps ; old-tap context], column tile c of Np1
//   B(c)       layer 2, column tile c of Np2
//   C0(g)      layer 3, the columns the mean needs for channel tile g (K = 1:
//              the mean; K = 3: three logits and three component means), and
//              y_hat = s + mean
//   C1(g)      layer 3, the scale columns of channel tile g, scale and index
//   H          (bf16, when enough slots are left) the hoisted layer-1 part
//              W1 psi + b1 of one task at a time, streaming its weights
// Each slice is held by kResRep workgroups (replicas) that take alternate
// tasks, two workgroups per compute unit.  A task of a role is one 16-row band (grid rows 16 beta .. 16 beta + 15 of
// image b) at one wavefront step t: the band's latents on wavefront t, at
// most one per grid row (Sec. III-A, Eq. 4: they are d-separated).  Every
// workgroup runs the tasks of its role in the same global order (steps, then
// images, then bands), computes its 16 x 16 (x the role's column tiles)
// output tile of the task with its register-resident weights, stores it with
// agent-coherent (sc1) stores and bumps the task's completion counter.  A
// task waits only for the bands it reads:
//   CTX(t, b, beta)  C0(t-lag) of bands beta and beta-1 (its taps are at
//                    least lag >= 2 steps old -- the parts before the last
//                    hold the rows furthest up, 4 steps old at the least
//                    with the 5x5 mask -- and lie at most R <= 3 rows up)
//   CTXL(t, b, beta) C0(t-2) of bands beta and beta-1, and every
//                    CTX(t, b, beta)
//   A(t, b, beta)    every CTXL(t, b, beta), C0(t-1) of bands beta and beta-1
//                    (the new taps, one step old)
//   B(t, b, beta)    every A(t, b, beta)
//   C0, C1(t, b, beta)  every B(t, b, beta)
//   H(k)             C0 of task k - 64 (it keeps a bounded lead); CTX (CTXL
//                    with one part) waits for H(k), so layer 1 follows it
// So bands of the upper grid rows run ahead of the lower ones, and no
// step-wide barrier exists.  Every (role, task) has its own counter, bumped
// once by each workgroup of the role when that workgroup's part of the task
// is stored; it is complete when it holds the role's workgroup count.  (A
// counter per band, reused by its successive tasks, would not do: workgroups
// that run ahead would make up for one that is still behind.)  Each counter
// has one slot per XCD class of the producers (256 bytes apart).  A workgroup
// finishes its tasks in order, so a complete task implies that the role's
// earlier tasks are complete too: waiting for the latest task a band had at
// or before a step covers all of the band's earlier steps.
// Every task writes its outputs (context parts, h1, h2) to buffers of its
// own, indexed by its position k in the global order, and y_hat is written
// once per latent, so no address is written twice in a call.  Producers store
// with write-through (sc1) stores.  The context roles and layer 3 bump the
// counter after their stores have landed, and their consumers read with
// ordinary cached loads: a line is first read, into an XCD's L2, only after
// its producer's counter was seen (the L2s start each launch empty of it), so
// the line the L2 keeps is current, and the workgroups of one XCD that read
// the same band share it there.  Layers 1 and 2 bump it as soon as every wave
// has issued its stores, without waiting for them to land: h1 and h2 are
// filled with an all-ones pattern before the launch (a NaN that lrelu of
// finite values never yields), and layers 2
// and 3 read them with agent-coherent (sc1) loads, which an XCD's L2 does not
// answer from a stale line, and load again until no value holds the pattern.
// A store's value is then seen by the first load after it lands, without the
// store acknowledgement and the counter bump in between.  This holds for fp32
// (kResChecked); in bf16 the decode came out slower (9.5 against 9.3 ms at
// 4K), so there layers 1 and 2 publish as the other roles do.
// Deadlock freedom: every dependency of a task comes earlier in the global
// order, and every workgroup runs its tasks in that order, so the earliest
// unfinished task can always run; the launch is cooperative, so all
// workgroups are resident.  Every wait has a wall-clock budget that records
// WF_E_TIMEOUT and makes every workgroup leave, so the grid always drains.
#include "wf_device.h"

namespace wf {

template <class P>
struct ResKb;
template <>
struct ResKb<PF32> {
    static constexpr int ctx = kResKbF32[0], a = kResKbF32[1], b = kResKbF32[2], c1 = kResKbF32[3],
                         c3 = kResKbF32[4], ctxl = kResKbF32[5];
};
template <>
struct ResKb<PBF16> {
    static constexpr int ctx = kResKbBf16[0], a = kResKbBf16[1], b = kResKbBf16[2], c1 = kResKbBf16[3],
                         c3 = kResKbBf16[4], ctxl = kResKbBf16[5];
};

// Wave-uniform copies of the argument blocks.  The role functions below are
// compiled out of line (each gets its own register allocation), and what they
// read through a reference to an argument block would otherwise count as
// per-lane data: every branch on it would become a divergent one.
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ float uni(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, v)));
}
template <class T>
__device__ __forceinline__ T* uni(T* p) {
    const unsigned long long v = reinterpret_cast<unsigned long long>(p);
    const unsigned lo = __builtin_amdgcn_readfirstlane((unsigned)v), hi = __builtin_amdgcn_readfirstlane((unsigned)(v >> 32));
    return reinterpret_cast<T*>(((unsigned long long)hi << 32) | lo);
}
// (Each copy starts as a plain copy, so a field missing from the lists below
// is still correct, only not marked uniform.)
__device__ __forceinline__ StepArgs uni_args(const StepArgs& x) {
    StepArgs a = x;
#define WF_U(f) a.f = uni(x.f)
    WF_U(H); WF_U(W); WF_U(M); WF_U(B); WF_U(K); WF_U(L); WF_U(lambda); WF_U(Np1); WF_U(Np2); WF_U(n3);
    WF_U(n_old); WF_U(ctx_parts); WF_U(R); WF_U(new_dx0); WF_U(slope); WF_U(group); WF_U(row_w); WF_U(gparts);
    WF_U(ec); WF_U(rowlat); WF_U(wp_all); WF_U(wp_hoist); WF_U(b_hoist); WF_U(wp_l1); WF_U(wp_new);
    WF_U(wp_new_lo); WF_U(wp_old); WF_U(wp2); WF_U(b2); WF_U(wp3); WF_U(b3); WF_U(table); WF_U(p1); WF_U(h1);
    WF_U(h2); WF_U(h2b); WF_U(ctxo); WF_U(ybf); WF_U(max_rows); WF_U(slots); WF_U(cp);
    for (int q = 0; q < kMaxRadius; ++q) WF_U(old_start[q]);
#undef WF_U
    return a;
}
__device__ __forceinline__ ResArgs uni_args(const ResArgs& x) {
    ResArgs r = x;
#define WF_U(f) r.f = uni(x.f)
    WF_U(per_slot); WF_U(parts); WF_U(pre_kb); WF_U(ctx_lag); WF_U(nrep); WF_U(nbands); WF_U(nbs); WF_U(cnt); WF_U(kbase); WF_U(steps); WF_U(ctx); WF_U(h1); WF_U(h2);
    WF_U(ytile);
    WF_U(err);
    WF_U(stamps); WF_U(ntasks); WF_U(stall); WF_U(hoist);
    for (int q = 0; q <= kResRoles; ++q) WF_U(first[q]);
#undef WF_U
    r.budget = ((long long)uni((int)(x.budget >> 32)) << 32) | (unsigned)uni((int)x.budget);
    r.stamps_cap = ((long long)uni((int)(x.stamps_cap >> 32)) << 32) | (unsigned)uni((int)x.stamps_cap);
    return r;
}

// Steps [t0, t1] during which band beta (grid rows 16 beta ..) holds latents.
__host__ __device__ __forceinline__ void band_span(int H, int W, int lam, int beta, int& t0, int& t1) {
    const int i0 = beta * kTile, i1 = min(H - 1, i0 + kTile - 1);
    t0 = lam * i0;
    t1 = lam * i1 + W - 1;
}
// Position in the global order of the latest task of band beta (image b) at
// a step <= s, or -1 when the band has none (beta < 0, or s before its first).
// kbase[t]: the position of step t's first task (kbase[T]: the number of
// tasks); steps[t]: step t's first band | its bands per image << 16 (tables,
// so that no wait divides by lambda).
template <class KB, class ST>
__host__ __device__ __forceinline__ int band_task_of(int H, int W, int lam, KB kbase, ST steps, int b, int beta,
                                                     int s) {
    if (beta < 0 || s < 0) return -1;
    int t0, t1;
    band_span(H, W, lam, beta, t0, t1);
    if (s < t0) return -1;
    const int t = s < t1 ? s : t1;
    const int st = steps[t];
    return kbase[t] + b * (st >> 16) + beta - (st & 0xFFFF);
}

// One wait: task k of `role` complete (nothing to wait for when k < 0).
struct ResWait {
    int role, k;
};
// The completions task k = (t, b, beta) of a role waits for (at most three;
// host and device: the roles take their waits from here, and the race checks
// of the test suite read the same ones through wf_plan_deps).  The old-tap
// context of step t reads y_hat of steps <= t-2 in the band's rows and the
// (up to R) rows above, the band above's at most: its latest tasks of step
// t-2 (each implies every earlier task of its band: C0(t') <- B(t') <- A(t')
// <- C0 of the band at t'-1).  The parts before the last hold the older taps
// (raster order, the rows furthest up first), so they wait for step t - lag
// with lag the smallest age among their taps (4 for the 5x5 mask's two
// parts); the last part waits for t - 2.  Layer 1 reads the two new taps,
// from step t-1 (the band's task and the band above's), and the task's
// context; layers 2 and 3 the layer before of the same task.
struct ResDeps {
    ResWait w[3];
};
// parts: the context's k-parts (CTX runs parts - 1 of them); lag: steps back
// to the youngest tap of those parts (>= 2); hoist: whether
// role RR_H computes the task's hoisted layer-1 part inside the launch.  The
// context waits for it (a free wait slot; layer 1, which reads it, waits for
// the context, so it follows).
template <class KB, class ST>
__host__ __device__ __forceinline__ ResDeps res_deps(int H, int W, int lam, KB kbase, ST steps, int role, int t, int b,
                                                     int beta, int k, int parts, int lag, int hoist) {
    ResDeps d{{{0, -1}, {0, -1}, {0, -1}}};
    switch (role) {
        case RR_CTX:
        case RR_CTXL: {
            const int s = role == RR_CTX ? t - lag : t - 2;
            d.w[0] = ResWait{RR_C0, band_task_of(H, W, lam, kbase, steps, b, beta, s)};
            d.w[1] = ResWait{RR_C0, band_task_of(H, W, lam, kbase, steps, b, beta - 1, s)};
            if (role == RR_CTXL && parts > 1) d.w[2] = ResWait{RR_CTX, k};   // the other parts, which it adds
            else if (hoist) d.w[2] = ResWait{RR_H, k};
            break;
        }
        case RR_A:
            d.w[0] = ResWait{RR_CTXL, k};
            d.w[1] = ResWait{RR_C0, band_task_of(H, W, lam, kbase, steps, b, beta, t - 1)};
            d.w[2] = ResWait{RR_C0, band_task_of(H, W, lam, kbase, steps, b, beta - 1, t - 1)};
            break;
        case RR_B:
            d.w[0] = ResWait{RR_A, k};
            break;
        case RR_H:   // reads only psi; paced to stay kResHoistLead tasks ahead of layer 3
            if (k >= kResHoistLead) d.w[0] = ResWait{RR_C0, k - kResHoistLead};
            break;
        default:   // RR_C0, RR_C1
            d.w[0] = ResWait{RR_B, k};
            break;
    }
    return d;
}
// The step table kbase, copied to LDS at the start of the launch: the waits
// of every task read it, and from LDS that costs no memory round trip.
__shared__ int res_kbase_lds[kResKbaseLds];
// and the per-step band table (first band | bands per image << 16)
__shared__ int res_steps_lds[kResKbaseLds];
// and the per-slot workgroup counts of the roles (the waits' targets)
__shared__ int res_per_slot_lds[kResRoles * kResRep * kXcds];

__device__ __forceinline__ ResDeps res_deps(const StepArgs& a, const ResArgs& r, int role, int t, int b, int beta,
                                            int k) {
    return res_deps(a.H, a.W, a.lambda, res_kbase_lds, res_steps_lds, role, t, b, beta, k, r.parts, r.ctx_lag,
                    r.hoist);
}

// Row r of band beta of image b at step t.
__device__ __forceinline__ Row band_row(const StepArgs& a, int b, int beta, int t, int r) {
    Row w;
    w.b = b;
    w.i = beta * kTile + r;
    w.j = t - a.lambda * w.i;
    w.valid = w.i < a.H && w.j >= 0 && w.j < a.W;
    w.lat = w.valid ? ((size_t)b * a.H + w.i) * a.W + w.j : 0;
    return w;
}

// The counters, the error word and the stamps are reached through global
// (address space 1) pointers and the bail flag through an LDS one: through
// generic pointers they would be flat accesses, and a flat access in flight
// makes the compiler wait for every load of a batch before its first MFMA
// (it cannot tell which counter a flat access is counted by).
typedef __attribute__((address_space(1))) unsigned gu32;
typedef __attribute__((address_space(1))) int gi32;
typedef __attribute__((address_space(3))) int li32;
template <class T>
__device__ __forceinline__ __attribute__((address_space(1))) T* glb(T* p) {
    return (__attribute__((address_space(1))) T*)p;
}

__device__ __forceinline__ gu32* res_slot(const ResArgs& r, int role, int k, int x) {
    return (gu32*)(r.cnt + (((size_t)role * r.ntasks + k) * kXcds + x) * kResSlotWords);
}

// Wave 0 polls up to three waits, eight lanes each (one per XCD class).  A
// wait longer than the budget, or an error recorded elsewhere, makes the
// workgroup leave (returns false).
__device__ __forceinline__ bool res_wait(const ResArgs& r, ResWait w0, ResWait w1, ResWait w2, int* bail) {
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x, i = lane >> 3, x = lane & (kXcds - 1);
        const ResWait w = i == 0 ? w0 : (i == 1 ? w1 : w2);
        unsigned tgt = 0;
        const gu32* p = (const gu32*)r.cnt;
        if (i < 3 && w.k >= 0) {
            // (one hoist workgroup per task, counting into class slot 0)
            const unsigned n =
                w.role == RR_H ? (x == 0 ? 1u : 0u)
                               : (unsigned)res_per_slot_lds[(w.role * kResRep + w.k % r.nrep) * kXcds + x];
            tgt = n + (unsigned)r.stall;
            p = res_slot(r, w.role, w.k, x);
        }
        int flag = 0;
        const long long t0 = wall_clock64();
        unsigned it = 0;
        while (true) {
            const unsigned v = tgt ? __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0u;
            if (__all(v >= tgt)) break;
            if ((++it & 63u) == 0) {
                if (__hip_atomic_load((gi32*)r.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) {
                    flag = 1;
                    break;
                }
                if (wall_clock64() - t0 > r.budget) {
                    if (lane == 0)
                        __hip_atomic_store((gi32*)r.err, kErrTimeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    flag = 1;
                    break;
                }
            }
            // (a longer sleep between polls thins the polls' memory traffic:
            // 4K 9.82 against 9.92 ms with sleep 1; 32 was slower again)
            __builtin_amdgcn_s_sleep(8);
        }
        if (lane == 0) *(li32*)bail = flag;
    }
    __syncthreads();
    return *(li32*)bail == 0;
}

// Count the task once every wave has issued its stores (their readers check
// the values; see the top of the file).
__device__ __forceinline__ void res_signal_issued(const ResArgs& r, int role, int k) {
    __builtin_amdgcn_s_barrier();
    if (threadIdx.x == 0)
        __hip_atomic_fetch_add(res_slot(r, role, k, blockIdx.x % kXcds), 1u, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
}

// Publish the task's stores (every wave's have landed) and count the task.
__device__ __forceinline__ void res_signal(const ResArgs& r, int role, int k) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0)
        __hip_atomic_fetch_add(res_slot(r, role, k, role == RR_H ? 0 : blockIdx.x % kXcds), 1u, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void res_stamp(const ResArgs& r, int k, int e) {
    if (r.stamps && threadIdx.x == 0) {
        const long long q = ((long long)k * gridDim.x + blockIdx.x) * 3 + e;
        if (q < r.stamps_cap) ((__attribute__((address_space(1))) long long*)r.stamps)[q] = wall_clock64();
    }
}

// The wave's share of a role's weights: k-blocks [kb0, kb0 + n) of NC column
// tiles ct0 + c * cstride of a packed panel with nkb k-blocks per column tile.
template <class P, int KB, int NC>
struct WSlice {
    typename P::B w[KB][NC];
    int kb0, n;
    __device__ __forceinline__ void split(int lo, int hi) {
        const int per = (hi - lo + kWaves - 1) / kWaves;
        kb0 = min(hi, lo + wave_id() * per);
        n = min(hi, kb0 + per) - kb0;
    }
    __device__ __forceinline__ void load(const void* panel, int nkb, int ct0, int cstride) {
        const typename P::B* p = static_cast<const typename P::B*>(panel) + (threadIdx.x & 63);
#pragma unroll
        for (int u = 0; u < KB; ++u)
#pragma unroll
            for (int c = 0; c < NC; ++c)
                w[u][c] = u < n ? p[((size_t)(ct0 + c * cstride) * nkb + kb0 + u) * 64] : typename P::B{};
    }
};

// Whether an fp32 activation operand holds the fill pattern of h1 / h2 (an
// all-ones word).
constexpr unsigned kResFill = 0xFFFFFFFFu;
template <class P>
constexpr bool kResChecked = !P::kBf16;
__device__ __forceinline__ bool holds_fill(const f4& v) {
    bool f = false;
#pragma unroll
    for (int j = 0; j < 4; ++j) f |= __builtin_bit_cast(unsigned, v[j]) == kResFill;
    return f;
}
// acc = the wave's k-blocks of a task's h1 / h2 tile (h, ncols columns) times
// its weight slice, read with agent-coherent loads until no value holds the
// fill pattern (the producers count their task before their stores land).
// The MFMAs run on every pass, each waiting only for its own load; the check
// follows them.  Past the wave's share the loads are masked (zeros) and the
// weights zero.  A pass count past the wall-clock budget records
// WF_E_TIMEOUT and ends the loop (the next wait then makes the workgroup
// leave).
template <class P, int KB, int NC>
__device__ __forceinline__ void wdot_checked(const WSlice<P, KB, NC>& s, const void* h, int ncols, bool valid,
                                             const ResArgs& r, f4 (&acc)[NC]) {
    const int n = __builtin_amdgcn_readfirstlane(s.n), kb0 = __builtin_amdgcn_readfirstlane(s.kb0);
    const long long t0 = wall_clock64();
    for (int it = 0;; ++it) {
        typename P::A av[KB];
#pragma unroll
        for (int u = 0; u < KB; ++u) av[u] = ld_tile<P, true>(h, 0, ncols, kb0 + u, valid && u < n);
        __builtin_amdgcn_sched_barrier(0);   // (all loads in flight before the first MFMA)
#pragma unroll
        for (int c = 0; c < NC; ++c) acc[c] = zero4();
#pragma unroll
        for (int u = 0; u < KB; ++u)
#pragma unroll
            for (int c = 0; c < NC; ++c) acc[c] = P::mma(av[u], s.w[u][c], acc[c]);
        bool seen = false;
#pragma unroll
        for (int u = 0; u < KB; ++u) seen |= holds_fill(av[u]);
        if (!__any(seen)) break;
        if ((it & 15) == 15 && wall_clock64() - t0 > r.budget) {
            if ((threadIdx.x & 63) == 0)
                __hip_atomic_store((gi32*)r.err, kErrTimeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            break;
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

// acc[c] += sum over the wave's k-blocks of A(kb) x W(kb, c), the
// activations loaded in batches of KBB k-blocks (each batch's loads issued
// before its first MFMA; one batch when KBB = KB).
template <class P, int KB, int NC, int KBB = KB, class LoadA>
__device__ __forceinline__ void wdot(const WSlice<P, KB, NC>& s, LoadA la, f4 (&acc)[NC]) {
    static_assert(KB % KBB == 0, "whole batches");
    // wave-uniform, in scalar registers: the guards below are then scalar
    // branches, and a batch's loads are all in flight before its first wait
    const int n = __builtin_amdgcn_readfirstlane(s.n), kb0 = __builtin_amdgcn_readfirstlane(s.kb0);
    if (n == KB) {
        // a full share: no guards, so each MFMA waits only for its own load
        // (with guards the compiler waits for every load before the first)
#pragma unroll
        for (int u0 = 0; u0 < KB; u0 += KBB) {
            typename P::A av[KBB];
#pragma unroll
            for (int u = 0; u < KBB; ++u) av[u] = la(kb0 + u0 + u);
            __builtin_amdgcn_sched_barrier(0);   // (all loads in flight before the first MFMA)
#pragma unroll
            for (int u = 0; u < KBB; ++u)
#pragma unroll
                for (int c = 0; c < NC; ++c) acc[c] = P::mma(av[u], s.w[u0 + u][c], acc[c]);
        }
        return;
    }
#pragma unroll
    for (int u0 = 0; u0 < KB; u0 += KBB) {
        if (u0 >= n) break;
        typename P::A av[KBB];
#pragma unroll
        for (int u = 0; u < KBB; ++u)
            if (u0 + u < n) av[u] = la(kb0 + u0 + u);
#pragma unroll
        for (int u = 0; u < KBB; ++u)
            if (u0 + u < n)
#pragma unroll
                for (int c = 0; c < NC; ++c) acc[c] = P::mma(av[u], s.w[u0 + u][c], acc[c]);
    }
}

// The same in two halves, for software pipelining: wload issues the loads of
// the wave's k-blocks into av, wmma consumes them.
template <class P, int KB, int NC, class LoadA>
__device__ __forceinline__ void wload(const WSlice<P, KB, NC>& s, LoadA la, typename P::A (&av)[KB]) {
    const int n = __builtin_amdgcn_readfirstlane(s.n), kb0 = __builtin_amdgcn_readfirstlane(s.kb0);
#pragma unroll
    for (int u = 0; u < KB; ++u)
        if (u < n) av[u] = la(kb0 + u);
}
template <class P, int KB, int NC>
__device__ __forceinline__ void wmma(const WSlice<P, KB, NC>& s, const typename P::A (&av)[KB], f4 (&acc)[NC]) {
    const int n = __builtin_amdgcn_readfirstlane(s.n);
#pragma unroll
    for (int u = 0; u < KB; ++u)
        if (u < n)
#pragma unroll
            for (int c = 0; c < NC; ++c) acc[c] = P::mma(av[u], s.w[u][c], acc[c]);
}

// The task after (t, b, beta) in the global order (t = T when there is none).
__device__ __forceinline__ void next_task(const StepArgs& a, int T, int& t, int& b, int& beta) {
    int i0, n;
    step_span(a.H, a.W, a.lambda, t, i0, n);
    if (beta < (i0 + n - 1) / kTile) {
        ++beta;
        return;
    }
    if (b + 1 < a.B) {
        ++b;
        beta = i0 / kTile;
        return;
    }
    b = 0;
    if (++t < T) {
        step_span(a.H, a.W, a.lambda, t, i0, n);
        beta = i0 / kTile;
    }
}

// Sum the four waves' partial tiles: afterwards lane l of wave w (< 4) holds
// in v[c] row 4 * (l / 16) + w, column l % 16 of tile c.
template <int NC>
__device__ __forceinline__ void wreduce(f4 (*red)[64], const f4 (&acc)[NC], float (&v)[NC]) {
    const int wave = wave_id(), lane = threadIdx.x & 63;
#pragma unroll
    for (int c = 0; c < NC; ++c) red[wave * NC + c][lane] = acc[c];
    __syncthreads();
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        v[c] = 0.0f;
#pragma unroll
        for (int w2 = 0; w2 < kWaves; ++w2) v[c] += red[w2 * NC + c][lane][wave];
    }
    __syncthreads();
}

// Visit the tasks (t, b, beta) of replica rep in the global order (position
// k with k % nrep == rep); body returns false to leave.
template <class F>
__device__ __forceinline__ void for_tasks(const StepArgs& a, int T, int rep, int nrep, F body) {
    int k = 0;
    for (int t = 0; t < T; ++t) {
        const int st = res_steps_lds[t], blo = st & 0xFFFF, bend = blo + (st >> 16);
        for (int b = 0; b < a.B; ++b)
            for (int beta = blo; beta < bend; ++beta, ++k)
                if (k % nrep == rep && !body(t, b, beta, k)) return;
    }
}

// Where the two new taps of one lane's row come from.  Both were decoded at
// the step before (they are one step old): the left tap (0, -1) in the same
// grid row, so row r of the band's task there; the upper tap (-1, new_dx0)
// in grid row i-1, so row r-1 of that task or, for r = 0, row 15 of the task
// of the band above.  Layer 3 keeps each task's y_hat as a 16 x M tile (tile
// order; bf16 as pairs), so a new-tap k-block is one 1 KB tile block read.
// Taps outside the grid (and rows without a latent) read zero.
struct NewSrc {
    size_t base[2];   // element offset of the source tile block of each tap
    bool ok[2];
};
// kself / kup: the band's task and the band above's task at step t-1 (-1: none).
template <class P>
__device__ __forceinline__ NewSrc new_src(const StepArgs& a, const Row& w, int kself, int kup) {
    const int rr = threadIdx.x & 15;
    NewSrc n;
#pragma unroll
    for (int tap = 0; tap < 2; ++tap) {
        const int ii = w.i + tap - 1, jj = w.j + (tap ? -1 : a.new_dx0);
        const int kt = (tap == 1 || rr > 0) ? kself : kup;
        const int row = tap == 1 ? rr : (rr + 15) & 15;
        n.ok[tap] = w.valid && ii >= 0 && jj >= 0 && jj < a.W && kt >= 0;
        // one task's tile: 16 x M values (bf16: pairs of halves)
        const size_t tb = (size_t)(kt >= 0 ? kt : 0) * kTile * a.M * (P::kBf16 ? 2 : 1);
        n.base[tap] = tb + tile_idx<P>(row, 0, a.M);
    }
    return n;
}

// The old-tap gathers of a context slice.  A wave's k-blocks [kb0, kb0 + n)
// cover at most kResSeg consecutive taps (segments); per task each lane
// computes one byte offset per segment, and k-block u of the wave then reads
// at off[seg(u)] + u * (bytes per k-block): the address arithmetic of a load
// is a select and an add.  Lanes whose tap lies outside the grid (or whose
// row has no latent) get an offset at or past the end of the buffer window,
// which the buffer unit answers with zeros.
constexpr int kResSeg = 4;
template <class P>
struct OldSrc {
    static constexpr int kKbBytes = P::kBf16 ? 128 : 64;   // one k-block of one row (bf16: hi and lo halves)
    // first wave k-block of segments 1-3 (uniform); the lane's byte offset of
    // segment 0 minus u * kKbBytes, and of segment q the difference to q - 1.
    // (Masked sums, not selects: the compiler turns a select chain over these
    // fields into a load through scratch memory.)
    int us1, us2, us3;
    int o0, d1, d2, d3;
    __device__ __forceinline__ int at(int u) const {
        return o0 + (d1 & -(int)(u >= us1)) + (d2 & -(int)(u >= us2)) + (d3 & -(int)(u >= us3)) + u * kKbBytes;
    }
};
// Row and column offset of old tap `tap` (taps in row-major order from row -R).
__device__ __forceinline__ void old_tap_dydx(const StepArgs& a, int tap, int& dy, int& dx) {
    static_assert(kMaxRadius == 3, "rows -3..0");
    const int row = tap < a.old_start[0] ? 0 : (tap < a.old_start[1] ? 1 : (tap < a.old_start[2] ? 2 : 3));
    const int first = row == 0 ? 0 : (row == 1 ? a.old_start[0] : (row == 2 ? a.old_start[1] : a.old_start[2]));
    dy = row - a.R;
    dx = tap - first - a.R;
}
// The wave's tap segments, the same for every task: their taps' offsets
// and first k-blocks, and each one's element offset within a latent.
struct OldTaps {
    int dy[kResSeg], dx[kResSeg], us[kResSeg], ke[kResSeg];
};
// kb0: the wave's first old-tap k-block (uniform).
template <class P>
__device__ __forceinline__ OldTaps old_taps(const StepArgs& a, int kb0) {
    const int M = a.M, tapkb = M / P::kK, kq = (threadIdx.x & 63) >> 4;
    const int tap0 = kb0 / tapkb;
    OldTaps o;
#pragma unroll
    for (int q = 0; q < kResSeg; ++q) {
        const int tap = min(tap0 + q, a.n_old - 1);
        // (past the wave's range when tap0 + q is past the taps)
        o.us[q] = q == 0 ? 0 : (tap0 + q) * tapkb - kb0;
        old_tap_dydx(a, tap, o.dy[q], o.dx[q]);
        // element of the lane's first channel of the tap's k-block kb0 within
        // the latent (may be negative for q > 0; the segment's own k-blocks
        // are not)
        if constexpr (P::kBf16)
            o.ke[q] = (kb0 - tap * tapkb) * 64 + kq * 8;    // pairs: 32 hi, 32 lo per k-block
        else
            o.ke[q] = (kb0 - tap * tapkb) * P::kK + kq * 4;
    }
    return o;
}
// w: the lane's row.
template <class P>
__device__ __forceinline__ OldSrc<P> old_src(const StepArgs& a, const Row& w, const OldTaps& ot) {
    const int M = a.M;
    int us[kResSeg], off[kResSeg];
#pragma unroll
    for (int q = 0; q < kResSeg; ++q) {
        us[q] = ot.us[q];
        const int ii = w.i + ot.dy[q], jj = w.j + ot.dx[q];
        const bool ok = w.valid && ii >= 0 && jj >= 0 && jj < a.W;
        const int lat = ok ? (w.b * a.H + ii) * a.W + jj : 0;
        const int e = lat * (P::kBf16 ? 2 * M : M) + ot.ke[q];
        off[q] = ok ? e * (P::kBf16 ? 2 : 4) : kBufBytes - us[q] * OldSrc<P>::kKbBytes;
    }
    OldSrc<P> o;
    o.us1 = us[1]; o.us2 = us[2]; o.us3 = us[3];
    o.o0 = off[0]; o.d1 = off[1] - off[0]; o.d2 = off[2] - off[1]; o.d3 = off[3] - off[2];
    return o;
}
// acc += the wave's old-tap k-blocks x its weight slice, all loads issued
// before the first MFMA.
template <class P, int KB, int NC>
__device__ __forceinline__ void wdot_old(const WSlice<P, KB, NC>& s, const void* src, OldSrc<P> os, f4 (&acc)[NC]) {
    const int n = __builtin_amdgcn_readfirstlane(s.n);
    const auto rs = rsrc(src);
    typename P::A av[KB];
    auto load = [&](int u) {
        const int off = os.at(u);
        if constexpr (P::kBf16)
            av[u] = b8x2{__builtin_bit_cast(b8, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0)),
                         __builtin_bit_cast(b8, __builtin_amdgcn_raw_buffer_load_b128(rs, off + 64, 0, 0))};
        else
            av[u] = __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
    };
    if (n == KB) {   // a full share: each MFMA waits only for its own load
#pragma unroll
        for (int u = 0; u < KB; ++u) load(u);
        // (keeps the scheduler from sinking each load next to its MFMA)
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < KB; ++u)
#pragma unroll
            for (int c = 0; c < NC; ++c) acc[c] = P::mma(av[u], s.w[u][c], acc[c]);
        return;
    }
#pragma unroll
    for (int u = 0; u < KB; ++u)
        if (u < n) load(u);
#pragma unroll
    for (int u = 0; u < KB; ++u)
        if (u < n)
#pragma unroll
            for (int c = 0; c < NC; ++c) acc[c] = P::mma(av[u], s.w[u][c], acc[c]);
}

// Element offset of context part `part` of task k (16 rows x 2M, tile order).
__device__ __forceinline__ size_t ctx_base(const StepArgs& a, const ResArgs& r, int k, int part) {
    return ((size_t)k * r.parts + part) * kTile * 2 * a.M;
}

// ---------------------------------------------------------------------------
// CTX(c, p) / CTXL(c): ctx[p][r][n] = sum over part p's old-tap k-blocks of
// taps x Wc for the NC column tiles of column group c; the last part (LAST)
// stores the sum over all parts.  A part's slice spans several column tiles
// so that each activation load feeds NC MFMAs (the activations of a task are
// the same for every column group, the weights differ).
template <class P, bool LAST>
__device__ __noinline__ void res_ctx(const StepArgs& a_in, const ResArgs& r_in, int T, int q, int rep, f4 (*red)[64],
                                     int* bail) {
    const StepArgs a = uni_args(a_in);
    const ResArgs r = uni_args(r_in);
    constexpr int KB = LAST ? ResKb<P>::ctxl : ResKb<P>::ctx;
    constexpr int NC = LAST ? kResCtxlNc : kResCtxNc;
    const int ncg = 2 * a.M / (kTile * NC);
    const int c = q % ncg, part = LAST ? r.parts - 1 : q / ncg;   // q: the slice
    const int lane = threadIdx.x & 63, kq = lane >> 4, wave = wave_id();
    const int nkb = a.n_old * a.M / P::kK, np = r.parts - 1;
    WSlice<P, KB, NC> s;
    if (LAST)
        s.split(r.pre_kb, nkb);
    else
        s.split(r.pre_kb * part / np, r.pre_kb * (part + 1) / np);
    s.load(a.wp_old, nkb, c * NC, 1);
    const int ro = kq * 4 + wave;
    const size_t pstride = (size_t)kTile * 2 * a.M;
    // the tap source, read once (not once per k-block): the call's
    // reconstruction (bf16: its pair copy)
    const void* src = P::kBf16 ? static_cast<const void*>(a.ybf) : static_cast<const void*>(uni(a.cp->y_hat));
    const int skb0 = __builtin_amdgcn_readfirstlane(s.kb0);
    const OldTaps ot = old_taps<P>(a, skb0);
    // the weight slice is in registers before the first task (else the
    // compiler, seeing its loads possibly in flight at every task, waits for
    // every load of each batch before its first MFMA)
    __builtin_amdgcn_s_waitcnt(0);
    for_tasks(a, T, rep, r.nrep, [&](int t, int b, int beta, int k) {
        res_stamp(r, k, 0);
        // the addresses depend on the task only: computed before the wait
        const size_t e = ctx_base(a, r, k, 0) + tile_idx<PF32>(ro, c * NC * kTile + (lane & 15), 2 * a.M);
        const Row w = band_row(a, b, beta, t, lane & 15);
        const OldSrc<P> os = old_src<P>(a, w, ot);
        const ResDeps dp = res_deps(a, r, LAST ? RR_CTXL : RR_CTX, t, b, beta, k);
        if (!res_wait(r, dp.w[0], dp.w[1], dp.w[2], bail)) return false;
        res_stamp(r, k, 1);
        // the other parts of these elements (the last part adds them; column
        // tile cc of the group is 256 elements of the tile order further)
        float prev[NC];
#pragma unroll
        for (int cc = 0; cc < NC; ++cc) prev[cc] = 0.0f;
        if constexpr (LAST) {
#pragma unroll
            for (int p2 = 0; p2 < kResMaxParts - 1; ++p2)
#pragma unroll
                for (int cc = 0; cc < NC; ++cc)
                    prev[cc] += ld1<false>(r.ctx, e + p2 * pstride + cc * 256, p2 < np);
        }
        f4 acc[NC];
#pragma unroll
        for (int cc = 0; cc < NC; ++cc) acc[cc] = zero4();
        // one load batch (the registers hold the weights and all of them)
        wdot_old<P, KB, NC>(s, src, os, acc);
        float v[NC];
        wreduce<NC>(red, acc, v);
#pragma unroll
        for (int cc = 0; cc < NC; ++cc) st1<true>(r.ctx, e + part * pstride + cc * 256, v[cc] + prev[cc]);
        res_signal(r, LAST ? RR_CTXL : RR_CTX, k);
        res_stamp(r, k, 2);
        return true;
    });
}

// A(c): h1 = lrelu(P1 + [new taps ; ctx] . [F_new ; W1b]) for column tile c.
template <class P>
__device__ __noinline__ void res_l1(const StepArgs& a_in, const ResArgs& r_in, int T, int c, int rep, f4 (*red)[64], int* bail) {
    const StepArgs a = uni_args(a_in);
    const ResArgs r = uni_args(r_in);
    const int lane = threadIdx.x & 63, kq = lane >> 4, wave = wave_id();
    const int M = a.M, ro = kq * 4 + wave, col = c * kTile + (lane & 15);
    const int kbn = kMaxNew * M / P::kK, kbc = 2 * M / P::kK, tapkb = M / P::kK;
    WSlice<P, ResKb<P>::a, 1> s;     // fp32: [F_new ; W1b]; bf16: F_new hi (new taps) or W1b (context)
    WSlice<P, ResKb<P>::a, 1> slo;   // bf16: F_new lo (new taps)
    // bf16: the new-tap and the context k-ranges are both 2M long; waves 0-1
    // take the new taps, waves 2-3 the context, so that each wave's loads are
    // one uniform batch
    const bool isnew = wave < kWaves / 2;
    if constexpr (P::kBf16) {
        const int lo = isnew ? 0 : kbn, hi = isnew ? kbn : kbn + kbc;
        const int per = (hi - lo + 1) / 2;
        s.kb0 = min(hi, lo + (wave & 1) * per);
        s.n = min(hi, s.kb0 + per) - s.kb0;
        slo.kb0 = s.kb0;
        slo.n = isnew ? s.n : 0;
        const typename P::B* ph = static_cast<const typename P::B*>(a.wp_new) + lane;
        const typename P::B* pl = static_cast<const typename P::B*>(a.wp_new_lo) + lane;
        const typename P::B* pc = static_cast<const typename P::B*>(a.wp_l1) + lane;
#pragma unroll
        for (int u = 0; u < ResKb<P>::a; ++u) {
            if (u >= s.n) continue;
            const int kb = s.kb0 + u;
            if (isnew) {
                s.w[u][0] = ph[((size_t)c * kbn + kb) * 64];
                slo.w[u][0] = pl[((size_t)c * kbn + kb) * 64];
            } else {
                s.w[u][0] = pc[((size_t)c * kbc + kb - kbn) * 64];
            }
        }
    } else {
        // fp32: every wave takes a quarter of the new-tap k-blocks (w[u],
        // u < KH) and a quarter of the context's (w[KH + u]), so that the
        // context half is computed as soon as the context is published and
        // only the new-tap half waits for the step before
        constexpr int KH = ResKb<P>::a / 2;
        const int hn = kbn / kWaves;
        const typename P::B* pw = static_cast<const typename P::B*>(a.wp_l1) + lane;
#pragma unroll
        for (int u = 0; u < KH; ++u) {
            s.w[u][0] = u < hn ? pw[((size_t)c * (kbn + kbc) + wave * hn + u) * 64] : zero4();
            s.w[KH + u][0] = u < hn ? pw[((size_t)c * (kbn + kbc) + kbn + wave * hn + u) * 64] : zero4();
        }
        s.kb0 = wave * hn;
        s.n = hn;
        slo.kb0 = 0;
        slo.n = 0;
    }
    const size_t h1s = (size_t)kTile * a.Np1 * 4;     // bytes of one task's h1
    // the weight slice is in registers before the first task (else the
    // compiler, seeing its loads possibly in flight at every task, waits for
    // every load of each batch before its first MFMA)
    __builtin_amdgcn_s_waitcnt(0);
    for_tasks(a, T, rep, r.nrep, [&](int t, int b, int beta, int k) {
        const int bs = b * r.nbands + beta;
        // the epilogue operand (hoisted before the launch) first
        const Row v = band_row(a, b, beta, t, ro);
        const size_t zq = v.lat * a.Np1 + col;
        // hoisted before the launch: loaded before the wait; else written in
        // this launch by role H (the context waited for it, and this role for
        // the context), with coherent loads, since P1 rows share lines
        // (both loads are issued in either case, one of them masked: a load
        // under a branch would keep the compiler from counting the batch's)
        float z = ld1<false>(a.p1, zq, v.valid && !r.hoist);
        res_stamp(r, k, 0);
        const ResDeps dp = res_deps(a, r, RR_A, t, b, beta, k);
        const int kself = dp.w[1].k, kup = dp.w[2].k;   // the new taps' tasks
        // (the addresses depend on the task only: computed before the wait)
        const Row w = band_row(a, b, beta, t, lane & 15);
        const NewSrc ns = new_src<P>(a, w, kself, kup);
        f4 acc[1] = {zero4()};
        if constexpr (!P::kBf16) {
            // the context half first (its one wait), then the new-tap half
            constexpr int KH = ResKb<P>::a / 2;
            const int hn = __builtin_amdgcn_readfirstlane(s.n), hk0 = __builtin_amdgcn_readfirstlane(s.kb0);
            const int ntap = hk0 >= tapkb;
            const size_t en = (ntap ? ns.base[1] : ns.base[0]) + (size_t)(hk0 - ntap * tapkb) * 256 + kq * 64;
            const size_t ec = ctx_base(a, r, k, r.parts - 1) + (size_t)hk0 * 256 + lane * 4;
            const int offn = (ntap ? ns.ok[1] : ns.ok[0]) ? (int)(en * 4) : kBufBytes;   // (past the window: zeros)
            const int offc = w.valid ? (int)(ec * 4) : kBufBytes;
            const ResWait none{0, -1};
            auto half = [&](const auto rs, int off, int u0) {
                f4 av[KH];
                if (hn == KH) {   // a full share: each MFMA waits only for its own load
#pragma unroll
                    for (int u = 0; u < KH; ++u)
                        av[u] = __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(rs, off + u * 1024, 0, 0));
                    __builtin_amdgcn_sched_barrier(0);   // (all loads in flight before the first MFMA)
#pragma unroll
                    for (int u = 0; u < KH; ++u) acc[0] = PF32::mma(av[u], s.w[u0 + u][0], acc[0]);
                } else {
#pragma unroll
                    for (int u = 0; u < KH; ++u)
                        if (u < hn)
                            av[u] = __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(rs, off + u * 1024, 0, 0));
#pragma unroll
                    for (int u = 0; u < KH; ++u)
                        if (u < hn) acc[0] = PF32::mma(av[u], s.w[u0 + u][0], acc[0]);
                }
            };
            if (!res_wait(r, dp.w[0], none, none, bail)) return false;
            half(rsrc(r.ctx), offc, KH);
            if (!res_wait(r, none, dp.w[1], dp.w[2], bail)) return false;
            res_stamp(r, k, 1);
            half(rsrc(r.ytile), offn, 0);
        } else {
            if (!res_wait(r, dp.w[0], dp.w[1], dp.w[2], bail)) return false;
            z += ld1<true>(a.p1, zq, v.valid && r.hoist);
            res_stamp(r, k, 1);
            const int sn = __builtin_amdgcn_readfirstlane(s.n), skb0 = __builtin_amdgcn_readfirstlane(s.kb0);
            if (isnew) {
                // the wave's k-blocks are those of one tap (two waves, two taps)
                const int tap = skb0 >= tapkb;
                const uint16_t* y = static_cast<const uint16_t*>(r.ytile);
                const size_t e = (tap ? ns.base[1] : ns.base[0]) + (size_t)(skb0 - tap * tapkb) * 1024 + kq * 128;
                const bool ok = tap ? ns.ok[1] : ns.ok[0];
                b8x2 av[ResKb<P>::a];
                auto load = [&](int u) { av[u] = b8x2{ld8h<false>(y, e + u * 1024, ok), ld8h<false>(y, e + u * 1024 + 512, ok)}; };
                auto mma = [&](int u) {
                    acc[0] = PBF16::mma(av[u], s.w[u][0], acc[0]);
                    acc[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[u].hi, slo.w[u][0], acc[0], 0, 0, 0);
                };
                if (sn == ResKb<P>::a) {   // a full share: each MFMA waits only for its own load
#pragma unroll
                    for (int u = 0; u < ResKb<P>::a; ++u) load(u);
                    __builtin_amdgcn_sched_barrier(0);   // (all loads in flight before the first MFMA)
#pragma unroll
                    for (int u = 0; u < ResKb<P>::a; ++u) mma(u);
                } else {
#pragma unroll
                    for (int u = 0; u < ResKb<P>::a; ++u)
                        if (u < sn) load(u);
#pragma unroll
                    for (int u = 0; u < ResKb<P>::a; ++u)
                        if (u < sn) mma(u);
                }
            } else {
                // the old-tap context (the last part's buffer holds the sum):
                // eight fp32 values per k-block, loaded first, split into
                // bf16 pairs afterwards
                const size_t e = ctx_base(a, r, k, r.parts - 1);
                f4 raw[ResKb<P>::a][2];
                auto load = [&](int u) {
                    const int c0 = (skb0 + u - kbn) * 32 + kq * 8;
                    raw[u][0] = ld4<false>(r.ctx, e + tile_idx<PF32>(lane & 15, c0, 2 * M), w.valid);
                    raw[u][1] = ld4<false>(r.ctx, e + tile_idx<PF32>(lane & 15, c0 + 4, 2 * M), w.valid);
                };
                if (sn == ResKb<P>::a) {   // a full share: each MFMA waits only for its own loads
#pragma unroll
                    for (int u = 0; u < ResKb<P>::a; ++u) load(u);
                    __builtin_amdgcn_sched_barrier(0);   // (all loads in flight before the first MFMA)
#pragma unroll
                    for (int u = 0; u < ResKb<P>::a; ++u)
                        acc[0] = PBF16::mma(split8(raw[u][0], raw[u][1]), s.w[u][0], acc[0]);
                } else {
#pragma unroll
                    for (int u = 0; u < ResKb<P>::a; ++u)
                        if (u < sn) load(u);
#pragma unroll
                    for (int u = 0; u < ResKb<P>::a; ++u)
                        if (u < sn) acc[0] = PBF16::mma(split8(raw[u][0], raw[u][1]), s.w[u][0], acc[0]);
                }
            }
        }
        float o[1];
        wreduce<1>(red, acc, o);
        st_tile<P, true>(static_cast<char*>(r.h1) + k * h1s, ro, a.Np1, col, lrelu(o[0] + z, a.slope));
        if constexpr (kResChecked<P>) res_signal_issued(r, RR_A, k);
        else res_signal(r, RR_A, k);
        res_stamp(r, k, 2);
        return true;
    });
}

// B(c): h2 = lrelu(W2 . h1 + b2) for column tile c.
template <class P>
__device__ __noinline__ void res_l2(const StepArgs& a_in, const ResArgs& r_in, int T, int c, int rep, f4 (*red)[64], int* bail) {
    const StepArgs a = uni_args(a_in);
    const ResArgs r = uni_args(r_in);
    const int lane = threadIdx.x & 63, kq = lane >> 4, wave = wave_id();
    const int ro = kq * 4 + wave, col = c * kTile + (lane & 15);
    const int nkb = a.Np1 / P::kK;
    WSlice<P, ResKb<P>::b, 1> s;
    s.split(0, nkb);
    s.load(a.wp2, nkb, c, 0);
    const float bias = a.b2[col];
    const size_t h1s = (size_t)kTile * a.Np1 * 4, h2s = (size_t)kTile * a.Np2 * 4;
    // the weight slice is in registers before the first task (else the
    // compiler, seeing its loads possibly in flight at every task, waits for
    // every load of each batch before its first MFMA)
    __builtin_amdgcn_s_waitcnt(0);
    for_tasks(a, T, rep, r.nrep, [&](int t, int b, int beta, int k) {
        const int bs = b * r.nbands + beta;
        res_stamp(r, k, 0);
        const ResDeps dp = res_deps(a, r, RR_B, t, b, beta, k);
        if (!res_wait(r, dp.w[0], dp.w[1], dp.w[2], bail)) return false;
        res_stamp(r, k, 1);
        const Row w = band_row(a, b, beta, t, lane & 15);
        const char* h1 = static_cast<const char*>(r.h1) + k * h1s;
        f4 acc[1] = {zero4()};
        if constexpr (kResChecked<P>) wdot_checked(s, h1, a.Np1, w.valid, r, acc);
        else wdot(s, [&](int kb) { return ld_tile<P, false>(h1, 0, a.Np1, kb, w.valid); }, acc);
        float o[1];
        wreduce<1>(red, acc, o);
        char* h2 = static_cast<char*>(r.h2) + k * h2s;
        st_tile<P, true>(h2, ro, a.Np2, col, lrelu(o[0] + bias, a.slope));
        if constexpr (kResChecked<P>) res_signal_issued(r, RR_B, k);
        else res_signal(r, RR_B, k);
        res_stamp(r, k, 2);
        return true;
    });
}

// C0(g) / C1(g): layer 3 of channel tile g and the parameter epilogue.
template <class P, int KC, bool MEAN>
__device__ __noinline__ void res_l3(const StepArgs& a_in, const ResArgs& r_in, int T, int g, int rep, f4 (*red)[64], const float* tab,
                       int* bail) {
    const StepArgs a = uni_args(a_in);
    const ResArgs r = uni_args(r_in);
    constexpr int NC = MEAN ? (KC == 1 ? 1 : 6) : KC;
    constexpr int KB = KC == 1 ? ResKb<P>::c1 : ResKb<P>::c3;
    const int lane = threadIdx.x & 63, kq = lane >> 4, wave = wave_id();
    const int M = a.M, G = M / kTile, ro = kq * 4 + wave, ch = g * kTile + (lane & 15);
    const int nkb = a.Np2 / P::kK;
    // first column tile of the role and the stride between its tiles
    const int ct0 = MEAN ? g : (KC == 1 ? G + g : 6 * G + g);
    WSlice<P, KB, NC> s;
    s.split(0, nkb);
    s.load(a.wp3, nkb, ct0, G);
    float bias[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) bias[c] = a.b3[(ct0 + c * G - g) * kTile + ch];
    const size_t h2s = (size_t)kTile * a.Np2 * 4;
    // the call's pointers, read once
    CallPtrs cpv;
    {
        const CallPtrs* cq = a.cp;
        cpv.sym = uni(cq->sym); cpv.y = uni(cq->y); cpv.sym_out = uni(cq->sym_out);
        cpv.y_hat = uni(cq->y_hat); cpv.mean = uni(cq->mean); cpv.scale = uni(cq->scale);
        cpv.weight = uni(cq->weight); cpv.cmean = uni(cq->cmean); cpv.idx = uni(cq->idx);
        cpv.encode = uni(cq->encode);
    }
    const CallPtrs* cp = &cpv;
    // the weight slice is in registers before the first task (else the
    // compiler, seeing its loads possibly in flight at every task, waits for
    // every load of each batch before its first MFMA)
    __builtin_amdgcn_s_waitcnt(0);
    for_tasks(a, T, rep, r.nrep, [&](int t, int b, int beta, int k) {
        const int bs = b * r.nbands + beta;
        const Row v = band_row(a, b, beta, t, ro);
        const size_t oq = v.lat * M + ch;
        // the symbol (or, encoding, y): both loads issued, one masked
        float sin = 0.0f;
        if constexpr (MEAN) {
            const float yv = ld1<false>(cp->y, oq, v.valid && cp->encode);
            const float sv = (float)__builtin_bit_cast(
                int32_t, ld1<false>(reinterpret_cast<const float*>(cp->sym), oq, v.valid && !cp->encode));
            sin = cp->encode ? yv : sv;
        }
        res_stamp(r, k, 0);
        const ResDeps dp = res_deps(a, r, MEAN ? RR_C0 : RR_C1, t, b, beta, k);
        if (!res_wait(r, dp.w[0], dp.w[1], dp.w[2], bail)) return false;
        res_stamp(r, k, 1);
        const Row w = band_row(a, b, beta, t, lane & 15);
        const char* h2 = static_cast<const char*>(r.h2) + k * h2s;
        f4 acc[NC];
#pragma unroll
        for (int c = 0; c < NC; ++c) acc[c] = zero4();
        if constexpr (kResChecked<P>) wdot_checked(s, h2, a.Np2, w.valid, r, acc);
        else wdot(s, [&](int kb) { return ld_tile<P, false>(h2, 0, a.Np2, kb, w.valid); }, acc);
        float o[NC];
        wreduce<NC>(red, acc, o);
#pragma unroll
        for (int c = 0; c < NC; ++c) o[c] += bias[c];
        if (v.valid) {
            if constexpr (!MEAN) {
                const float t0 = tab[0];
#pragma unroll
                for (int kk = 0; kk < KC; ++kk) {
                    const float sg = o[kk] > t0 ? o[kk] : t0;
                    const size_t q2 = (v.lat * KC + kk) * M + ch;
                    glb(cp->scale)[q2] = sg;
                    glb(cp->idx)[q2] = scale_index(tab, a.L, sg);
                }
            } else {
                float mu;
                if constexpr (KC == 1) {
                    mu = o[0];
                } else {
                    const float mx = fmaxf(o[0], fmaxf(o[1], o[2]));
                    float ex[3], den = 0.0f;
#pragma unroll
                    for (int kk = 0; kk < 3; ++kk) {
                        ex[kk] = expf(o[kk] - mx);
                        den += ex[kk];
                    }
                    mu = 0.0f;
#pragma unroll
                    for (int kk = 0; kk < 3; ++kk) {
                        const float wk = ex[kk] / den;
                        const size_t q2 = (v.lat * 3 + kk) * M + ch;
                        glb(cp->weight)[q2] = wk;
                        glb(cp->cmean)[q2] = o[3 + kk];
                        mu += wk * o[3 + kk];
                    }
                }
                float sv;
                if (cp->encode) {
                    sv = rintf(sin - mu);
                    glb(cp->sym_out)[oq] = (int32_t)sv;
                } else {
                    sv = sin;
                }
                glb(cp->mean)[oq] = mu;
                st1<true>(cp->y_hat, oq, sv + mu);
                if constexpr (P::kBf16) st_pair_row<true>(a.ybf, v.lat * 2 * M, ch, sv + mu);
                // the task's tile of y_hat, the next step's new taps
                st_tile<P, true>(static_cast<char*>(r.ytile) + (size_t)k * kTile * M * 4, ro, M, ch, sv + mu);
            }
        }
        res_signal(r, MEAN ? RR_C0 : RR_C1, k);
        res_stamp(r, k, 2);
        return true;
    });
}

// H(h): the hoisted part of layer 1, P1 = b_hoist + W1[:, :2M] . psi, for the
// latents of every task k with k mod nh = h, all Np1 columns: each wave takes
// every fourth group of four column tiles over the whole K (no cross-wave
// reduction), streaming the weights, and the results go out with coherent
// stores.  The task's context waits for it.  It waits only to stay a fixed
// number of tasks ahead of layer 3, so that its products spread over the
// decode instead of crowding the first steps' compute units.
template <class P>
__device__ __noinline__ void res_hoist(const StepArgs& a_in, const ResArgs& r_in, int T, int h, int nh, int* bail) {
    const StepArgs a = uni_args(a_in);
    const ResArgs r = uni_args(r_in);
    using A = typename P::A;
    using Bw = typename P::B;
    constexpr int NC = 4, KB = 8;
    const int lane = threadIdx.x & 63, kq = lane >> 4, wave = wave_id();
    const int nct = a.Np1 / kTile, nkb = 2 * a.M / P::kK, M = a.M;
    const float* psi = uni(a.cp->psi);
    // (global, not generic: flat loads would keep the compiler from counting
    // the batch's loads one by one)
    const __attribute__((address_space(1))) Bw* wp = (const __attribute__((address_space(1))) Bw*)a.wp_hoist + lane;
    for_tasks(a, T, h, nh, [&](int t, int b, int beta, int k) {
        res_stamp(r, k, 0);
        const ResDeps dp = res_deps(a, r, RR_H, t, b, beta, k);
        if (!res_wait(r, dp.w[0], dp.w[1], dp.w[2], bail)) return false;
        res_stamp(r, k, 1);
        const Row w = band_row(a, b, beta, t, lane & 15);   // the lane's operand row
        size_t olat[4];                                      // its epilogue rows
        bool ov[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const Row v = band_row(a, b, beta, t, kq * 4 + q);
            olat[q] = v.lat;
            ov[q] = v.valid;
        }
        auto la = [&](int kb) -> A {
            if constexpr (P::kBf16) {
                const size_t q = w.lat * 2 * M + kb * 32 + kq * 8;
                return split8(ld4<false>(psi, q, w.valid), ld4<false>(psi, q + 4, w.valid));
            } else {
                return ld4<false>(psi, w.lat * 2 * M + kb * kTile + kq * 4, w.valid);
            }
        };
        for (int c0 = wave * NC; c0 < nct; c0 += kWaves * NC) {
            f4 acc[NC];
#pragma unroll
            for (int c = 0; c < NC; ++c) acc[c] = zero4();
            for (int kc = 0; kc < nkb; kc += KB) {
                A av[KB];
                Bw bv[KB][NC];
#pragma unroll
                for (int u = 0; u < KB; ++u) {
                    const int kk = min(kc + u, nkb - 1);
                    av[u] = la(kk);
#pragma unroll
                    for (int c = 0; c < NC; ++c) bv[u][c] = wp[((size_t)min(c0 + c, nct - 1) * nkb + kk) * 64];
                }
#pragma unroll
                for (int u = 0; u < KB; ++u)
                    if (kc + u < nkb)
#pragma unroll
                        for (int c = 0; c < NC; ++c) acc[c] = P::mma(av[u], bv[u][c], acc[c]);
            }
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                if (c0 + c >= nct) continue;
                const int n = (c0 + c) * kTile + (lane & 15);
                const float bias = a.b_hoist[n];
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (ov[q]) st1<true>(a.p1, olat[q] * a.Np1 + n, acc[c][q] + bias);
            }
        }
        res_signal(r, RR_H, k);
        res_stamp(r, k, 2);
        return true;
    });
}

// Two workgroups per compute unit (each wave at most 256 registers).
template <class P, int KC>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_resident(
    StepArgs a, ResArgs r, int T) {
    __shared__ f4 red[kWaves * kResMaxNc][64];
    __shared__ float tab[kMaxTable];
    __shared__ int bail;
    for (int l = threadIdx.x; l < a.L; l += blockDim.x) tab[l] = a.table[l];
    for (int l = threadIdx.x; l <= T; l += blockDim.x) res_kbase_lds[l] = r.kbase[l];   // (T < kResKbaseLds)
    for (int l = threadIdx.x; l < T; l += blockDim.x) res_steps_lds[l] = r.steps[l];
    for (int l = threadIdx.x; l < kResRoles * kResRep * kXcds; l += blockDim.x) res_per_slot_lds[l] = r.per_slot[l];
    __syncthreads();
    // (selects, not a loop: a runtime index into the argument block would
    // copy it to scratch memory)
    const int g = blockIdx.x;
    const int role = (g >= r.first[1]) + (g >= r.first[2]) + (g >= r.first[3]) + (g >= r.first[4]) +
                     (g >= r.first[5]) + (g >= r.first[6]);
    const int q = g - (role == 0   ? 0
                       : role == 1 ? r.first[1]
                       : role == 2 ? r.first[2]
                       : role == 3 ? r.first[3]
                       : role == 4 ? r.first[4]
                       : role == 5 ? r.first[5]
                                   : r.first[6]);
    if (role == RR_H) {   // one task in every nh, each workgroup its own
        res_hoist<P>(a, r, T, q, r.first[7] - r.first[6], &bail);
        return;
    }
    // slices of the role (its workgroups are nrep replicas of each)
    const int nsl = ((role == 0   ? r.first[1]
                      : role == 1 ? r.first[2] - r.first[1]
                      : role == 2 ? r.first[3] - r.first[2]
                      : role == 3 ? r.first[4] - r.first[3]
                      : role == 4 ? r.first[5] - r.first[4]
                                  : r.first[6] - r.first[5])) / r.nrep;
    const int sl = q % nsl, rep = q / nsl;
    // Layer 1 issues ahead of the other workgroup on its compute unit (a
    // context part or a layer-3 half): its tasks are short and every step's
    // chain runs through them. Raising layer 2 or 3 as well, or the context
    // above layers 2-3, made the decode slower.
    if (role == RR_A) __builtin_amdgcn_s_setprio(2);
    switch (role) {
    case RR_CTX:
        res_ctx<P, false>(a, r, T, sl, rep, red, &bail);
        break;
    case RR_CTXL:
        res_ctx<P, true>(a, r, T, sl, rep, red, &bail);
        break;
    case RR_A: res_l1<P>(a, r, T, sl, rep, red, &bail); break;
    case RR_B: res_l2<P>(a, r, T, sl, rep, red, &bail); break;
    case RR_C0: res_l3<P, KC, true>(a, r, T, sl, rep, red, tab, &bail); break;
    default: res_l3<P, KC, false>(a, r, T, sl, rep, red, tab, &bail); break;
    }
}

__global__ void k_res_fill(unsigned* p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = kResFill;
}

// Zero the n counter slots (only their first words).
__global__ void k_res_zero(unsigned* p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i * kResSlotWords] = 0u;
}

static const void* resident_fn(const Plan& p) {
    if (p.precision == WF_BF16)
        return p.K == 1 ? (const void*)k_resident<PBF16, 1> : (const void*)k_resident<PBF16, 3>;
    return p.K == 1 ? (const void*)k_resident<PF32, 1> : (const void*)k_resident<PF32, 3>;
}

template <class T>
static int res_alloc(Plan& p, T** dst, size_t n) {
    hipError_t e = hipMalloc((void**)dst, n * sizeof(T));
    if (e != hipSuccess) return fail(WF_E_NOMEM, std::string("hipMalloc: ") + hipGetErrorString(e));
    p.owned.push_back(*dst);
    return WF_OK;
}

static int ceil_div(int a, int b) { return (a + b - 1) / b; }

// kbase[t] = the position of step t's first task in the global order (t, b,
// band), kbase[T] = the number of tasks; steps[t] = step t's first band |
// its bands per image << 16; returns the number of tasks.
static long long res_kbase(const Plan& p, std::vector<int>& kbase, std::vector<int>& steps) {
    kbase.assign(p.T + 1, 0);
    steps.assign(p.T, 0);
    long long tasks = 0;
    for (int t = 0; t < p.T; ++t) {
        int i0, nn;
        step_span(p.H, p.W, p.lambda, t, i0, nn);
        const int blo = i0 / kTile, nb = (i0 + nn - 1) / kTile - blo + 1;
        kbase[t] = (int)tasks;
        steps[t] = blo | nb << 16;
        tasks += (long long)p.B * nb;
    }
    kbase[p.T] = (int)tasks;
    return tasks;
}

// The split of the old taps between the context parts: the last part takes
// the taps (raster order) from the first one of age 2 -- the steps between
// producer and consumer -- on, or as many of the last taps as its slice holds
// when those are more; the parts before it take the rest.  Returns their
// k-blocks (pre_kb) and the smallest age among them (lag: 3 or more when the
// taps of age 2 are all in the last part, else 2).
void res_ctx_split(const Plan& p, int& pre_kb, int& lag) {
    const bool bf = p.precision == WF_BF16;
    const int kk = bf ? 32 : 16, tapkb = p.M / kk;
    const int last_max = kWaves * (bf ? kResKbBf16[5] : kResKbF32[5]) / tapkb;   // taps a last-part slice holds
    std::vector<int> ages;
    for (int k = 0; k < p.ntaps; ++k) {
        if (p.dy[k] < 0 && p.dx[k] >= p.W) continue;   // never in the grid (left out of the old taps)
        const int age = p.lambda * (-p.dy[k]) - p.dx[k];
        if (age >= 2) ages.push_back(age);
    }
    const int n = (int)ages.size();
    int pre = n;
    for (int u = 0; u < n; ++u)
        if (ages[u] == 2) {
            pre = u;
            break;
        }
    pre = std::max(pre, n - last_max);
    lag = 1 << 30;
    for (int u = 0; u < pre; ++u) lag = std::min(lag, ages[u]);
    if (lag == 1 << 30) lag = 2;
    pre_kb = pre * tapkb;
}

// The tasks and waits of a plan's geometry (host only, for the race checks):
// per task in the global order {t, b, band, then for each role its three
// waits as (role, task)}.
int resident_deps(const Plan& p, std::vector<int32_t>& out) {
    int pre_kb, lag2;
    res_ctx_split(p, pre_kb, lag2);
    std::vector<int> kbase, steps;
    const long long tasks = res_kbase(p, kbase, steps);
    if (tasks > INT32_MAX / 64) return fail(WF_E_UNSUPPORTED, "too many resident tasks");
    out.clear();
    int k = 0;
    for (int t = 0; t < p.T; ++t) {
        int i0, n;
        step_span(p.H, p.W, p.lambda, t, i0, n);
        for (int b = 0; b < p.B; ++b)
            for (int beta = i0 / kTile; beta <= (i0 + n - 1) / kTile; ++beta, ++k) {
                const int32_t head[3] = {t, b, beta};
                out.insert(out.end(), head, head + 3);
                for (int role = 0; role < kResRoles; ++role) {
                    // (as planned on a device with room for the context
                    // parts before the last and, for bf16, the in-launch
                    // hoist)
                    const ResDeps d = res_deps(p.H, p.W, p.lambda, kbase.data(), steps.data(), role, t, b, beta, k,
                                               pre_kb > 0 ? 2 : 1, lag2, p.precision == WF_BF16 ? 1 : 0);
                    for (int i = 0; i < 3; ++i) {
                        out.push_back(d.w[i].k >= 0 ? d.w[i].role : -1);
                        out.push_back(d.w[i].k);
                    }
                }
            }
    }
    return WF_OK;
}

int build_resident(Plan& p) {
    const StepArgs& a = p.args;
    ResArgs& r = p.res;
    const bool bf = p.precision == WF_BF16;
    const int* kb = bf ? kResKbBf16 : kResKbF32;
    // The roles read data written earlier in the launch with ordinary cached
    // loads, which is safe only if no 128-byte line holds data of two tasks:
    // a line fetched with a latent that another task writes later would stay
    // stale in the reader's L2.  Per-task buffers are whole lines; y_hat rows
    // (M floats) are whole lines when M is a multiple of 32.
    if (p.M % 32 != 0) return fail(WF_E_UNSUPPORTED, "resident driver: M must be a multiple of 32");
    const int kk = bf ? 32 : 16;
    const int M = p.M, G = M / kTile, ncg = 2 * M / (kTile * kResCtxNc), ncgl = 2 * M / (kTile * kResCtxlNc);
    const int nkb_old = a.n_old * M / kk;
    int pre_kb, lag;
    res_ctx_split(p, pre_kb, lag);
    // every wave's share of every slice must fit its registers
    if (ceil_div((kMaxNew * M + 2 * M) / kk, kWaves) > kb[1] || ceil_div(p.Np1 / kk, kWaves) > kb[2] ||
        ceil_div(p.Np2 / kk, kWaves) > kb[p.K == 1 ? 3 : 4] || ceil_div(nkb_old - pre_kb, kWaves) > kb[5] ||
        (2 * M) % (kTile * kResCtxNc) != 0)
        return fail(WF_E_UNSUPPORTED, "resident driver: a weight slice exceeds the register budget (M too large)");
    int cus = 0, dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return fail(WF_E_HIP, std::string("device query: ") + hipGetErrorString(e));
    if (p.cu_limit > 0 && p.cu_limit < cus) cus = p.cu_limit;
    const int crit = p.Np1 / kTile + p.Np2 / kTile + 2 * G;
    const int slots = kResRep * cus;   // two workgroups per compute unit
    // the fewest parts before the last whose slices fit the registers
    int np = 0;
    if (pre_kb > 0)
        for (np = 1; ceil_div(ceil_div(pre_kb, np), kWaves) > kb[0];) ++np;
    if (np + 1 > kResMaxParts) return fail(WF_E_UNSUPPORTED, "resident driver: the old-tap context needs too many parts");
    auto need = [&](int n_) { return kResRep * (crit + ncg * n_ + ncgl); };
    if (need(np) > slots)
        return fail(WF_E_UNSUPPORTED, "resident driver: " + std::to_string(need(np)) + " workgroups for " +
                                          std::to_string(slots) + " slots");
    // fp32: spare slots take more context parts (shorter context tasks);
    // bf16: they compute the hoisted layer-1 part in the launch (4K: 9.74 ms
    // with 68 such workgroups and the fewest parts, 9.87 with 48, 11.0 with
    // 28 and two more parts)
    while (!bf && np > 0 && need(np + 1) <= slots && np + 2 <= kResMaxParts && pre_kb / (np + 1) >= kWaves) ++np;
    const int parts = np + 1;
    // a wave's old-tap k-blocks must lie in at most kResSeg taps
    {
        const int tapkb = M / kk;
        for (int q = 0; q < parts; ++q) {
            const int lo = q < np ? pre_kb * q / np : pre_kb, hi = q < np ? pre_kb * (q + 1) / np : nkb_old;
            const int per = ceil_div(hi - lo, kWaves);
            for (int wv = 0; wv < kWaves; ++wv) {
                const int k0 = std::min(hi, lo + wv * per), k1 = std::min(hi, k0 + per);
                if (k1 > k0 && (k1 - 1) / tapkb - k0 / tapkb + 1 > kResSeg)
                    return fail(WF_E_UNSUPPORTED, "resident driver: a context slice spans too many taps (M too small)");
            }
        }
    }
    r.parts = parts;
    r.pre_kb = pre_kb;
    r.ctx_lag = lag;
    r.nrep = kResRep;
    const int n[RR_H] = {ncg * np, ncgl, p.Np1 / kTile, p.Np2 / kTile, G, G};
    r.first[0] = 0;
    for (int k = 0; k < RR_H; ++k) r.first[k + 1] = r.first[k] + kResRep * n[k];
    // bf16: the slots left over compute the hoisted layer-1 part inside the
    // launch, one task each in turn (4K: 9.74 against 10.19 ms with the hoist
    // kernel before the launch).  fp32: the kernel before the launch (the
    // in-launch hoist's fp32 products slow the roles they share compute units
    // with: 14.6-14.9 against 14.0 ms, measured before the context parts were
    // re-blocked), as with too few spare slots.
    const int spare = slots - r.first[RR_H];
    const int nh = bf && spare >= kResMinHoist ? spare : 0;
    r.first[kResRoles] = r.first[RR_H] + nh;
    r.hoist = nh > 0 ? 1 : 0;
    const int grid = r.first[kResRoles];
    int per_slot[kResRoles * kResRep * kXcds] = {};
    for (int k = 0; k < RR_H; ++k)
        for (int g = r.first[k]; g < r.first[k + 1]; ++g) {
            const int h = (g - r.first[k]) / n[k];   // the workgroup's replica
            ++per_slot[(k * kResRep + h) * kXcds + g % kXcds];
        }
    int* d_per = nullptr;
    int rc;
    if ((rc = res_alloc(p, &d_per, kResRoles * kResRep * kXcds)) != WF_OK) return rc;
    e = hipMemcpy(d_per, per_slot, sizeof(per_slot), hipMemcpyHostToDevice);
    if (e != hipSuccess) return fail(WF_E_HIP, std::string("hipMemcpy: ") + hipGetErrorString(e));
    r.per_slot = d_per;
    r.nbands = ceil_div(p.H, kTile);
    r.nbs = p.B * r.nbands;
    const size_t nbs = (size_t)r.nbs;
    if (p.T + 1 > kResKbaseLds)
        return fail(WF_E_UNSUPPORTED, "resident driver: more than " + std::to_string(kResKbaseLds - 1) + " wavefront steps");
    std::vector<int> kbase, steps;
    const long long tasks = res_kbase(p, kbase, steps);
    r.ntasks = (int)tasks;
    int *d_kbase = nullptr, *d_steps = nullptr;
    if ((rc = res_alloc(p, &d_kbase, kbase.size())) != WF_OK) return rc;
    e = hipMemcpy(d_kbase, kbase.data(), kbase.size() * sizeof(int), hipMemcpyHostToDevice);
    if (e != hipSuccess) return fail(WF_E_HIP, std::string("hipMemcpy: ") + hipGetErrorString(e));
    if ((rc = res_alloc(p, &d_steps, steps.size())) != WF_OK) return rc;
    e = hipMemcpy(d_steps, steps.data(), steps.size() * sizeof(int), hipMemcpyHostToDevice);
    if (e != hipSuccess) return fail(WF_E_HIP, std::string("hipMemcpy: ") + hipGetErrorString(e));
    r.kbase = d_kbase;
    r.steps = d_steps;
    if ((rc = res_alloc(p, &r.cnt, (size_t)kResRoles * tasks * kXcds * kResSlotWords)) != WF_OK) return rc;
    // one output buffer per task (no address is written twice in a call);
    // each is read through raw buffer loads and must fit their window
    const size_t nt = (size_t)tasks;
    const size_t ctx_n = nt * parts * kTile * 2 * M, h1_n = nt * kTile * p.Np1, h2_n = nt * kTile * p.Np2;
    if (std::max(ctx_n, std::max(h1_n, h2_n)) * 4 >= (size_t)kBufBytes)
        return fail(WF_E_UNSUPPORTED, "resident driver: per-task buffers exceed the 2 GiB buffer window");
    if ((rc = res_alloc(p, &r.ctx, ctx_n)) != WF_OK) return rc;
    float *h1 = nullptr, *h2 = nullptr, *yt = nullptr;
    if ((rc = res_alloc(p, &h1, h1_n)) != WF_OK) return rc;
    if ((rc = res_alloc(p, &h2, h2_n)) != WF_OK) return rc;
    if ((rc = res_alloc(p, &yt, nt * kTile * M)) != WF_OK) return rc;
    r.h1 = h1;
    r.h2 = h2;
    r.ytile = yt;
    r.err = p.d_err;
    r.budget = p.spin_budget;
    // one workgroup per compute unit, all resident at once
    int per_cu = 0;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, resident_fn(p), kThreads, 0);
    if (e != hipSuccess) return fail(WF_E_HIP, std::string("occupancy query: ") + hipGetErrorString(e));
    if (per_cu < kResRep) return fail(WF_E_UNSUPPORTED, "resident kernel: two workgroups per CU do not fit");
    p.grid = grid;
    return WF_OK;
}

int enqueue_resident(Plan& p, hipStream_t stream) {
    ResArgs r = p.res;
    r.stamps = p.stamps;
    r.stamps_cap = p.stamps_cap;
    r.budget = p.spin_budget;
    r.stall = p.stall;
    const size_t ncnt = (size_t)kResRoles * r.ntasks * kXcds;
    hipLaunchKernelGGL(k_res_zero, dim3(1024), dim3(256), 0, stream, r.cnt, ncnt);
    // fp32: h1 and h2 to the fill pattern their readers check for
    if (p.precision != WF_BF16) {
        hipLaunchKernelGGL(k_res_fill, dim3(2048), dim3(256), 0, stream, static_cast<unsigned*>(r.h1),
                           (size_t)r.ntasks * kTile * p.Np1);
        hipLaunchKernelGGL(k_res_fill, dim3(2048), dim3(256), 0, stream, static_cast<unsigned*>(r.h2),
                           (size_t)r.ntasks * kTile * p.Np2);
    }
    if (!r.hoist) {
        int rc = enqueue_hoist(p, stream);
        if (rc != WF_OK) return rc;
    }
    StepArgs a = p.args;
    int T = p.T;
    void* args[] = {&a, &r, &T};
    hipError_t e = hipLaunchCooperativeKernel(resident_fn(p), dim3(p.grid), dim3(kThreads), args, 0, stream);
    if (e != hipSuccess) return fail(WF_E_HIP, std::string("cooperative launch: ") + hipGetErrorString(e));
    return WF_OK;
}

}  // namespace wf
