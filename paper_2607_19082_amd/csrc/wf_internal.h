// Internal declarations shared by the host plan code and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "wf.h"

namespace wf {

constexpr int kMaxTaps = 24;         // the 7x7 causal mask
constexpr int kTaps5x5 = 12;         // the 5x5 causal mask
constexpr int kMaxRadius = 3;
// rANS (entropy coding of the symbols): probabilities in units of 2^-16, a
// 64-bit state in [2^31, 2^63) renormalised by 32-bit words, and per level a
// table of the symbol at the start of each 16-slot bucket.
constexpr int kEcPrecBits = 16;
constexpr int kEcLutShift = 4;
constexpr int kEcLut = 1 << (kEcPrecBits - kEcLutShift);
constexpr int kEcMaxSupport = 16383;   // support half-width bound (symbol indices fit 16 bits)
// the 3-component mixture's coder: sixteenths of a symbol, offsets within
// +-2^14 of them, weights summing to 2^12, CDFs scaled by 2^20, at most 2^15
// coded symbols per latent
constexpr int kMixFine = 16, kMixQmax = 1 << 14, kMixCdfBits = 20, kMixMaxSymbols = 1 << 15;
// device error word values
constexpr int kErrTimeout = 1, kErrStream = 2, kErrCapacity = 3;
constexpr int kMaxNew = 2;           // taps written by the immediately preceding step
constexpr int kTile = 16;            // MFMA tile edge (rows and columns)
constexpr int kJobWaves = 4;         // waves of one job's workgroup
constexpr int kCtxPartsF32 = 6;      // k-parts of the old-tap context product, fp32 operands
constexpr int kCtxPartsBf16 = 3;     // the same, bf16 operands
constexpr int kDfCtxParts = 2;       // the same for the dataflow driver (its context jobs run
                                     // in a pool of their own, where fewer, longer jobs pay)
constexpr int kCtxPartsMax = kCtxPartsF32 > kCtxPartsBf16 ? kCtxPartsF32 : kCtxPartsBf16;
static_assert(kDfCtxParts <= kCtxPartsMax, "context k-parts exceed the buffer");
constexpr int kColsF32 = 1;          // column tiles of one job, fp32 operands
constexpr int kColsBf16 = 2;         // the same, bf16 operands
constexpr int kMaxTable = 256;
constexpr int kXcds = 8;             // accelerator complex dies of an MI355X
constexpr int kBarrierWords = 4096;  // barrier counters of the persistent driver
constexpr int kBufBytes = 0x7fff0000; // window of a raw buffer access (arrays must fit)
constexpr int kDfSlotWords = 16;     // dataflow counter slots: one per 64 bytes

// Job kinds of the dataflow driver (see wf_dataflow.hip).
enum JobKind { JK_CTX = 0, JK_CTXL = 1, JK_A = 2, JK_B = 3, JK_C0 = 4, JK_C1 = 5, kJobKinds = 6 };

// Column tiles ct in [lo, hi) with ct % 8 == x.
__host__ __device__ __forceinline__ int cnt_range(int lo, int hi, int x) {
    auto upto = [](int n, int x) { return n > x ? (n - x + kXcds - 1) / kXcds : 0; };
    return upto(hi, x) - upto(lo, x);
}

// Dataflow driver state passed to its kernel: the per-XCD-class job lists
// (job code {t, kind | part << 4 | rt << 8 | ct << 16}) and the counters.
// Counter group (t, kind, rt) counts the finished jobs of that step, kind and
// row tile; rt = nrt_max holds the step's total (kept for JK_C0 and JK_C1).
// Each group has one slot per XCD class, bumped by the jobs of that class.
// Two pools of workgroups take jobs from separate lists: workgroups
// [0, ncrit) the critical chain (N, A, B, C0, C1), the others the old-tap
// context (CTX, CTXL), so that a critical job never waits behind context work
// queued in its workgroup's list.
struct DfArgs {
    const int2* jobs;
    int off[2 * kXcds + 1]; // list x (critical) is jobs[off[x], off[x+1]), list 8 + x (context) follows
    int ncrit;              // workgroups of the critical pool (a multiple of 8)
    unsigned* cnt;
    size_t cnt_words;
    int nrt_max;            // 16-row tiles of the widest step
    long long* stamps;      // optional trace: 3 wall-clock ticks per job (see wf_plan_trace)
    long long stamps_cap;
    int stall;              // test hook: every wait's target one more than it can reach
};

// Resident driver (see wf_resident.hip): roles of its workgroups, in this
// order of workgroup indices.
enum ResRole { RR_CTX = 0, RR_CTXL = 1, RR_A = 2, RR_B = 3, RR_C0 = 4, RR_C1 = 5, RR_H = 6, kResRoles = 7 };
// Weight k-blocks one wave holds in registers per column tile, by role
// (fp32 k-blocks of 16, bf16 k-blocks of 32); a plan whose slices need more
// is not supported by that driver.
// per-wave k-blocks of a slice: context part (kResCtxNc column tiles), layer 1,
// layer 2, layer 3 (K = 1), layer 3 (K = 3), last context part (kResCtxlNc tiles)
constexpr int kResKbF32[6] = {6, 20, 17, 14, 8, 10};
constexpr int kResKbBf16[6] = {6, 10, 9, 7, 4, 10};
constexpr int kResCtxNc = 4;       // column tiles of a context part's slice (64 of the 2M columns)
constexpr int kResCtxlNc = 2;      // column tiles of a last-part slice
constexpr int kResMaxNc = 6;        // column tiles of one layer-3 role (K = 3: 3 logits + 3 means)
constexpr int kResMaxParts = 12;    // k-parts of the old-tap context (the last one included)
// Resident completion counters: one slot every 256 bytes.  With the slots
// 64 bytes apart (four in a 256-byte block) the 4K decode took 10.29 ms
// fp32 / 9.19 bf16, 256 bytes apart 9.92 / 8.45, 512 or 1024 no better;
// 32 bytes apart, or packed, 12.4-16.5 ms.
constexpr int kResSlotWords = 64;
constexpr int kResRep = 2;          // replicas of every weight slice (they take alternate tasks)
constexpr int kResKbaseLds = 4096;  // largest T + 1 of a resident plan (its step table sits in LDS)
constexpr int kResMinHoist = 8;     // fewest spare workgroups that compute the hoisted layer-1 part in the launch
constexpr int kResHoistLead = 64;   // tasks by which that part runs ahead of layer 3

struct ResArgs {
    int first[kResRoles + 1];   // workgroups [first[r], first[r+1]) play role r
    const int* per_slot;        // [kResRoles][kResRep][8]: workgroups of role r, replica h, in XCD class x
    int parts;                  // k-parts of the old-tap context: parts - 1 split the old taps before the
                                // first one of age 2 (raster order; k-blocks [0, pre_kb)) evenly, the
                                // last one (CTXL) holds the rest, [pre_kb, n_old M / kK)
    int pre_kb;
    int ctx_lag;                // steps between a CTX task and the C0 tasks it waits for: the smallest
                                // age of the old taps before pre_kb (CTXL waits for step t - 2)
    int nrep;                   // replicas of each weight slice: workgroup q of a role with n slices holds
                                // slice q % n and runs the tasks k with k % nrep == q / n.  CTX slices are
                                // (column tile, part 0 .. parts-2), CTXL slices the column tiles of the
                                // last part, which adds the other parts in
    int nbands;                 // 16-row bands per image (ceil(H / 16)); band slot bs = b * nbands + band
    int nbs;                    // B * nbands
    unsigned* cnt;              // [kResRoles][ntasks][8] counter slots, kResSlotWords words apart
    const int* kbase;           // [T + 1] position of each step's first task in the global order
    const int* steps;           // [T] first band of each step | its bands per image << 16
    float* ctx;                 // [ntasks][parts] x (16 x 2M) old-tap context k-parts of each task
    void* h1;                   // [ntasks] x (16 x Np1) layer-1 output of each task (tile order)
    void* h2;                   // [ntasks] x (16 x Np2) layer-2 output of each task
    void* ytile;                // [ntasks] x (16 x M) y_hat of each task's latents (tile order; bf16: pairs),
                                // the source of the next step's new taps
    int* err;
    long long budget;
    long long* stamps;          // optional trace: 3 wall-clock ticks per task and workgroup
    long long stamps_cap;
    int ntasks;                 // tasks of every workgroup (band visits of all steps and images)
    int stall;                  // test hook: every wait's target one more than it can reach
    int hoist;                  // 1: the workgroups of role RR_H compute the hoisted layer-1 part
                                // per task inside the launch (else a kernel before it does)
};

// Set the calling thread's error message and return `code`.
int fail(int code, const std::string& msg);

// Pointers of one decode/encode call.  They live in plan-owned device memory
// and are written by a one-thread kernel before the step kernels run, so a
// captured graph of step kernels serves every call.
struct CallPtrs {
    const float* psi;       // [B][H][W][2M]
    const int32_t* sym;     // decode input
    const float* y;         // encode input
    int32_t* sym_out;       // encode output; decode from streams: the decoded symbols
    float *y_hat, *mean, *scale, *weight, *cmean;
    int32_t* idx;
    int encode;
    // Decode from rANS streams (StepArgs::ec): the caller's words, the plan's
    // per-stream decoder state and tables, and the device error word.
    const uint32_t* bits;
    uint64_t* ec_x;         // [B*H*M] decoder states
    uint32_t *ec_pos, *ec_end;   // [B*H*M] next word, one past the stream's last
    const int32_t* ec_n;    // [L] support half-width per level
    const int32_t* ec_base; // [L] first cumulative entry per level
    const uint32_t* ec_cum; // cumulative frequencies
    const uint64_t* ec_lut; // [L][kEcLut] per slot bucket: its first slot's symbol u, cum[u], cum[u + 1]
    // the 3-component mixture (K = 3): per level l the half-width X_l of its
    // integer CDF on sixteenths of a symbol, its first entry, and the CDFs
    const int32_t* mix_X;   // [L]
    const int32_t* mix_base;// [L]
    const uint32_t* mix_G;  // G_l(x), x = -X_l..X_l, at mix_base[l] + x + X_l
    int* err;
};

// Plan constants passed by value to every step kernel.
//
// Taps are split by age.  A tap (dy,dx) of the latent decoded at step t was
// written at step t - delta with delta = lambda*(-dy) - dx.  Only the "new"
// taps (delta = 1) are gathered on the critical path of step t; the context
// sum over the "old" taps (delta >= 2) of step t+1's latents only needs
// y_hat of steps <= t-1, so it is computed during step t, off the critical
// path, in k-parts.
//
// Layer 1 of step t reads [new taps (kMaxNew*M) ; old-tap context (2M)]
// against [W1[:, 2M:] . Wc[new taps] ; W1[:, 2M:]] (the new taps' conv and the
// context half of layer 1 are both linear, so their product is folded at plan
// time; the context bias is folded into the hoisted part).  With bf16
// operands the folded block is formed from the bf16 weights and kept as a
// bf16 pair (wp_new + wp_new_lo), the rest of the panel is wp_l1.
//
// Packed weights (wp_*) hold 16-byte lane operands per (column tile, k-block):
// fp32 k-blocks of 16, bf16 k-blocks of 32.  Np1, Np2 are d1, d2 rounded up to
// a whole k-block and a whole column group (kColsF32 / kColsBf16 tiles).
struct StepArgs {
    int H, W, M, B, K, L, lambda;
    int Np1, Np2, n3;
    int n_old;              // old taps (the new ones are kMaxNew)
    int ctx_parts;          // k-parts of the old-tap context product (per driver, precision)
    // Tap geometry, as scalars so that kernels compute a tap's offset without
    // indexing memory.  The mask has radius R (rows -R..0).  Old taps are
    // tap-major by row; old_start[q] is the first old tap of row -R + q + 1
    // (a sentinel above any tap for rows past 0), the first of row -R is 0;
    // each row's run starts at dx = -R and is contiguous.  New taps:
    // (-1, new_dx0) and (0, -1).
    int R;
    int old_start[kMaxRadius];
    int new_dx0;
    float slope;
    // Context approximation (groups of `group` wavefronts; 1 = exact decode).
    // A "step" is then a group; its rows are listed in rowlat (latent indices,
    // from StepRows::r0), its context is the product over all taps (raster
    // mask order: row_w taps in each of rows -R..-1 from dx = -R, then the R
    // taps (0,-R)..(0,-1)) with same-group taps filled, in gparts k-parts.
    int group, row_w, gparts;
    int ec;                 // 1: phase C decodes each symbol from its rANS stream
    const int* rowlat;      // nullptr: rows of wavefront t by grid row
    const void* wp_all;     // packed Wc over all taps, channel-chunk-major k   [2M/16][(n_old+2)*M/kb]
    const void* wp_hoist;   // packed W1[:, :2M]                           [Np1/16][2M/kb]
    const float* b_hoist;   // b1 + W1[:, 2M:] . bc (bf16: the bf16 W1)    [Np1]
    const void* wp_l1;      // fp32: packed [W1b.Wc[new] ; W1b]            [Np1/16][(2M + 2M)/16]
                            // bf16: packed W1b                            [Np1/16][2M/32]
    const void* wp_new;     // bf16: packed F_new = W1b . Wc[new], hi half [Np1/16][2M/32]
    const void* wp_new_lo;  // bf16: the same, lo half
    const void* wp_old;     // packed Wc over the old taps                 [2M/16][n_old*M/kb]
    const void* wp2;        // packed W2                                   [Np2/16][Np1/kb]
    const float* b2;        // [Np2]
    const void* wp3;        // packed W3                                   [n3/16][Np2/kb]
    const float* b3;        // [n3]
    const float* table;     // [L]
    float* p1;              // [B*H*W][Np1] hoisted layer-1 part
    // per-step activations, max_rows x n in MFMA operand order (tile_idx):
    void* h1;               // n = Np1, fp32 or bf16 pairs
    void* h2;               // n = Np2, fp32 or bf16 pairs (even steps)
    void* h2b;              // the same for odd steps (dataflow driver; else == h2)
    float* ctxo;            // [2][parts] x (n = 2M) old-tap context k-parts, by step parity
    uint16_t* ybf;          // bf16: [B*H*W][M/32][2][32] y_hat as bf16 pairs (tap source)
    int max_rows;           // rows of the widest step, rounded up to 16
    int slots;              // workgroups resident at once (jobs of one round)
    const CallPtrs* cp;
};

struct Plan {
    // description
    int H, W, M, B, K, d1, d2, n3, mask, precision, driver, L;
    float slope;
    // schedule
    int lambda, T, ntaps;
    int group;                           // wavefronts per decoding step (1: exact)
    int steps;                           // decoding steps: T, or ceil(T / group)
    std::vector<int> g_r0, g_n;          // grouped decode: rows of each group in rowlat
    int dy[kMaxTaps], dx[kMaxTaps];
    std::vector<int32_t> step_of;        // [H*W]
    int max_rows;
    int Np1, Np2;                        // d1, d2 rounded up to a whole k-block
    int nph;                             // phases per step: 3 (fp32) or 4 (bf16)
    StepArgs args;                       // device pointers filled in
    // device memory owned by the plan
    int device = 0;
    std::vector<void*> owned;
    CallPtrs* d_call = nullptr;
    int* d_err = nullptr;
    // persistent driver
    unsigned* d_bar = nullptr;
    int grid = 0;
    long long spin_budget = 100000000;   // wall-clock ticks (100 MHz): 1 s
    int stall = 0;                        // test hook: every in-launch wait unreachable
    int cu_limit = 0;                     // plan for at most this many CUs (0: all)
    long long* stamps = nullptr;         // optional barrier trace
    long long stamps_cap = 0;
    // dataflow driver
    DfArgs df{};
    // resident driver
    ResArgs res{};
    // graph driver
    hipStream_t cap_stream = nullptr;
    hipGraph_t graph = nullptr;
    hipGraphExec_t graph_exec = nullptr;
    // entropy coding (rANS): tables, decoder states, encoder scratch and, for
    // the graph driver, the graph of the decode from streams
    int ec = 0;
    int32_t *ec_n = nullptr, *ec_base = nullptr;
    uint32_t* ec_cum = nullptr;
    uint64_t* ec_lut = nullptr;
    uint64_t* ec_x = nullptr;
    uint32_t *ec_pos = nullptr, *ec_end = nullptr, *ec_len = nullptr, *ec_words = nullptr;
    int32_t *mix_X = nullptr, *mix_base = nullptr;   // K = 3: the mixture's level CDFs
    uint32_t* mix_G = nullptr;
    hipGraph_t graph_ec = nullptr;
    hipGraphExec_t graph_exec_ec = nullptr;
};

// Enqueue the kernels of one call after its pointers were published to
// p.d_call (used directly by the stream driver and captured by the graph
// driver).
int enqueue_steps(Plan& p, hipStream_t stream, bool ec = false);
// The same with explicit plan constants (the workspace pointers of `a` may
// point elsewhere than the plan's own, see wf_decode_noalloc).
int enqueue_steps_with(const Plan& p, const StepArgs& a, hipStream_t stream, bool ec = false);
// Publish a call's pointers to the block at dst.
int enqueue_set_call_at(CallPtrs* dst, const CallPtrs& c, hipStream_t stream);
// entropy coding (wf_ec.hip)
int build_ec(Plan* p, const float* scale_table, int L);
int enqueue_ec_init(Plan& p, const uint32_t* bits, int64_t n_words, const uint32_t* offsets, hipStream_t stream);
// (the encode's outputs give each symbol's parameters: idx, and for K = 3
// weight, comp_mean and mean)
int enqueue_ec_encode(Plan& p, const int32_t* sym, const wf_out& out, uint32_t* bits, int64_t cap,
                      uint32_t* offsets, hipStream_t stream);
// Publish the call's pointers to p.d_call on `stream`.
int enqueue_set_call(Plan& p, const CallPtrs& c, hipStream_t stream);
// The pre-loop product of the hyperprior half of layer 1.
int enqueue_hoist(Plan& p, hipStream_t stream);
// Persistent driver: grid size (checked co-residency) and one call.
int persistent_grid(Plan& p, int* grid);
int enqueue_persistent(Plan& p, hipStream_t stream);
// Dataflow driver: job lists of the plan, and one call.
// (order: optionally each list entry's position in the global order)
int build_dataflow(Plan& p, std::vector<int2>& lists, DfArgs& d, std::vector<int>* order = nullptr);
// Job lists and waits of a plan's geometry, flattened (host only; wf_plan_deps).
int dataflow_deps(Plan& p, std::vector<int32_t>& out);
int enqueue_dataflow(Plan& p, hipStream_t stream);
const void* dataflow_fn(const Plan& p);
// Resident driver: roles and buffers of the plan, and one call.
int build_resident(Plan& p);
// Tasks and waits of a plan's geometry, flattened (host only; wf_plan_deps).
int resident_deps(const Plan& p, std::vector<int32_t>& out);
int enqueue_resident(Plan& p, hipStream_t stream);
// Grid of a cooperative kernel: two workgroups per CU when they fit, else one.
int coop_grid(Plan& p, const void* fn, int* grid);
// Latency floor of one dependent step hop (see wf_measure_floor).
int measure_floor(Plan& p, float* node_us, float* barrier_us);

}  // namespace wf
