// Device code shared by the per-step kernels and the persistent kernel: the
// MFMA tile engine and the work of the phases of a wavefront step.
//
// fp32 operands, step t (Sec. III-C), three phases:
//   phase A  h1 = lrelu(P1 + [new taps ; ctx_old(t)] . [F_new ; W1b])
//   phase B  h2 = lrelu(W2 . h1 + b2)
//   phase C  o  = W3 . h2 + b3 -> mean / scale / index, y_hat = s + mean
// with P1 = b1 + W1b . bc + W1[:, :2M] . psi hoisted before the loop,
// W1b = W1[:, 2M:], F_new = W1b . Wc[new taps] folded at plan time, and
// ctx_old(t+1) = Wc[old taps] . y_hat[old taps] for the latents of step t+1
// (its inputs were all written by step t-1 or earlier).
//
// bf16 operands (weights rounded to bf16, every activation carried as a pair
// of bf16 values hi = bf16(x), lo = bf16(x - hi), fp32 accumulation): the same
// three phases; F_new is formed from the bf16 weights and carried as a bf16
// pair as well, so the fold adds no coarse rounding, and phase C also keeps the
// pair form of y_hat for the tap gathers.  Pair arrays: see tile_idx and
// st_pair_row.
// The last of the P::kParts k-parts of ctx_old(t+1) adds the others in and
// runs in phase C; the other parts ride along with the phases of step t,
// spread to even out their work (see step_work).
//
// Every product runs on MFMA: fp32 v_mfma_f32_16x16x4f32 (four chained per
// 16 values of k) or bf16 v_mfma_f32_16x16x32_bf16.  Each wave issues all
// operand loads of its k-range before its first MFMA, and the epilogue
// operands are fetched before the products.  Jobs are placed XCD-aware:
// block b runs on XCD b % 8, and each column tile of a weight matrix is always
// computed on the same XCD, which then streams only its slice of the weights.
//
// COH selects how data produced by other workgroups of the same launch is
// accessed: with COH the activations, the reconstruction and the old-tap
// context are written and read with agent-coherent (sc1) buffer operations, so
// the persistent kernel needs no cache flush between its phases.
#pragma once

#include "wf_internal.h"

namespace wf {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 b8 __attribute__((ext_vector_type(8)));
struct b8x2 {   // eight activation values as bf16 pairs
    b8 hi, lo;
};

constexpr int kWaves = kJobWaves;      // waves per workgroup; they split a tile's k-blocks
constexpr int kThreads = 64 * kWaves;
constexpr int kSc1 = 16;   // cache-policy bits of an agent-coherent buffer access
constexpr int kMaxPhases = 4;
constexpr int kMaxC = kColsF32 > kColsBf16 ? kColsF32 : kColsBf16;   // most column tiles of one job (rows of the reduction buffer: kWaves * kMaxC)

// Phases of a step, in order: PH_A..PH_C (the grouped decode: PH_GX, PH_GA, PH_B, PH_C).
enum { PH_A = 1, PH_B = 2, PH_C = 3, PH_GX = 4, PH_GA = 5 };   // PH_G*: grouped decode

__device__ __forceinline__ f4 mfma_k16(f4 a, f4 b, f4 acc) {
    // Lane l supplies A[l%16][4*(l/16)+q] and B[4*(l/16)+q][l%16] for the q-th
    // instruction: the four instructions together sum over 16 values of k.
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, b.x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, b.y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, b.z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, b.w, acc, 0, 0, 0);
    return acc;
}

// Operand precisions.  A k-block is the k extent of one lane operand of a
// 16x16 tile (16 values for fp32, 32 for bf16); lane l supplies A row l%16 /
// B column l%16 at the k-group l/16 of the block, 4 (fp32) or 8 (bf16)
// consecutive k, so one 16-byte load per lane per k-block feeds B (and A, or
// each half of a bf16 activation pair).  The products only need A and B to
// use the same k order, which the packing of the weights and the activation
// loads share.  A bf16 k-block is two MFMAs: weights times hi, times lo.
struct PF32 {
    using A = f4;   // activation operand
    using B = f4;   // weight operand
    static constexpr int kK = 16;
    static constexpr bool kBf16 = false;
    static constexpr int kFirst = PH_A;
    static constexpr int kC = kColsF32;               // column tiles of one job (A loaded once for all)
    static constexpr int kParts = kCtxPartsF32;       // k-parts of the old-tap context
    static constexpr int kKbw = 10;                   // k-blocks a wave loads before its MFMAs
    static constexpr int kL3Kbw1 = 16, kL3Kbw3 = 4;   // the same for l3 (K = 1, 3)
    __device__ static __forceinline__ f4 mma(A a, B b, f4 acc) { return mfma_k16(a, b, acc); }
};
struct PBF16 {
    using A = b8x2;
    using B = b8;
    static constexpr int kK = 32;
    static constexpr bool kBf16 = true;
    static constexpr int kFirst = PH_A;
    static constexpr int kC = kColsBf16;
    static constexpr int kParts = kCtxPartsBf16;
    static constexpr int kKbw = 10;
    static constexpr int kL3Kbw1 = 8, kL3Kbw3 = 3;
    __device__ static __forceinline__ f4 mma(A a, B b, f4 acc) {
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.hi, b, acc, 0, 0, 0);
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.lo, b, acc, 0, 0, 0);
    }
};

__device__ __forceinline__ float lrelu(float v, float s) { return v >= 0.0f ? v : s * v; }

// The wave's index in its workgroup, as a wave-uniform value: k-ranges and
// tap geometry derived from it then live in scalar registers and scalar
// branches, not in per-lane arithmetic under exec masks.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

__device__ __forceinline__ f4 zero4() { return f4{0.0f, 0.0f, 0.0f, 0.0f}; }

// fp32 -> bf16, round to nearest even (v_cvt_pk_bf16_f32 in the default mode).
__device__ __forceinline__ uint16_t bf16_bits(float v) { return __builtin_bit_cast(uint16_t, (__bf16)v); }
__device__ __forceinline__ float bf16_value(uint16_t h) { return __builtin_bit_cast(float, (unsigned)h << 16); }

__device__ __forceinline__ b8 to_b8(f4 a, f4 b) {
    b8 r;
    r[0] = (__bf16)a.x; r[1] = (__bf16)a.y; r[2] = (__bf16)a.z; r[3] = (__bf16)a.w;
    r[4] = (__bf16)b.x; r[5] = (__bf16)b.y; r[6] = (__bf16)b.z; r[7] = (__bf16)b.w;
    return r;
}

// Eight fp32 values as bf16 pairs (x - hi is exact in fp32).
__device__ __forceinline__ b8x2 split8(f4 a, f4 b) {
    const b8 hi = to_b8(a, b);
    const f4 ha{(float)hi[0], (float)hi[1], (float)hi[2], (float)hi[3]};
    const f4 hb{(float)hi[4], (float)hi[5], (float)hi[6], (float)hi[7]};
    return b8x2{hi, to_b8(a - ha, b - hb)};
}

// Raw buffer resource over [p, p + kBufBytes): accesses at or past kBufBytes
// return zero.  Every base pointer used here is the same for the whole wave;
// reading it from the first lane keeps the descriptor in scalar registers.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p) {
    const unsigned long long v = reinterpret_cast<unsigned long long>(p);
    const unsigned lo = __builtin_amdgcn_readfirstlane((unsigned)v);
    const unsigned hi = __builtin_amdgcn_readfirstlane((unsigned)(v >> 32));
    void* u = reinterpret_cast<void*>(((unsigned long long)hi << 32) | lo);
    return __builtin_amdgcn_make_buffer_rsrc(u, (short)0, kBufBytes, 0x00020000);
}

// Activation loads go through raw buffer instructions: an invalid element
// (row past the step, tap outside the grid) is given an offset past the end
// of the 2 GiB window, which the buffer unit answers with zeros.  The loaders
// are therefore branch-free and a wave's loads can all be in flight at once.
// With COH the access is agent-coherent (sc1), for data written by other
// workgroups of the same launch.  (The buffer builtins move raw 32-bit words:
// bit casts, not conversions.)
// kOob lies past the window under either range rule (offset >= size, or
// offset + access size > size).
constexpr int kOob = 0x7ffffff0;
static_assert(kOob >= kBufBytes + 16, "the sentinel offset must be out of range");

template <bool COH>
__device__ __forceinline__ f4 ld4(const float* base, size_t idx, bool ok = true) {
    const int off = ok ? (int)(idx * 4) : kOob;
    return __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(rsrc(base), off, 0, COH ? kSc1 : 0));
}
template <bool COH>
__device__ __forceinline__ float ld1(const float* base, size_t idx, bool ok = true) {
    const int off = ok ? (int)(idx * 4) : kOob;
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc(base), off, 0, COH ? kSc1 : 0));
}
// eight bf16 values at element idx of a bf16 array
template <bool COH>
__device__ __forceinline__ b8 ld8h(const uint16_t* base, size_t idx, bool ok = true) {
    const int off = ok ? (int)(idx * 2) : kOob;
    return __builtin_bit_cast(b8, __builtin_amdgcn_raw_buffer_load_b128(rsrc(base), off, 0, COH ? kSc1 : 0));
}
template <bool COH>
__device__ __forceinline__ void st1(float* base, size_t idx, float v) {
    if (COH)
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), rsrc(base), (int)(idx * 4), 0, kSc1);
    else
        base[idx] = v;
}
template <bool COH>
__device__ __forceinline__ void st1h(uint16_t* base, size_t idx, uint16_t h) {
    if (COH)
        __builtin_amdgcn_raw_buffer_store_b16(h, rsrc(base), (int)(idx * 2), 0, kSc1);
    else
        base[idx] = h;
}

// The per-step activation arrays (h1, h2, the bf16 context vector and the
// fp32 old-tap context parts) are kept in MFMA operand order: for 16-row tile
// rt and k-block kb of rows of n values, the 64 lanes' 16-byte A operands lie
// next to each other (fp32: 1 KB per block; bf16 pairs: 1 KB of hi halves,
// then 1 KB of lo halves), so every A load is one contiguous 1 KB.  tile_idx
// is the element index of (row r, column c) (bf16: of its hi half; the lo
// half is 512 elements further).
template <class P>
__device__ __forceinline__ size_t tile_idx(int r, int c, int n) {
    if constexpr (P::kBf16)
        return ((size_t)(r >> 4) * (n >> 5) + (c >> 5)) * 1024 + (((c & 31) >> 3) * 16 + (r & 15)) * 8 + (c & 7);
    else
        return ((size_t)(r >> 4) * (n >> 4) + (c >> 4)) * 256 + (((c & 15) >> 2) * 16 + (r & 15)) * 4 + (c & 3);
}
// A operand of k-block kb of row tile rt.
template <class P, bool COH>
__device__ __forceinline__ typename P::A ld_tile(const void* base, int rt, int n, int kb, bool ok) {
    const int lane = threadIdx.x & 63;
    if constexpr (P::kBf16) {
        const uint16_t* h = static_cast<const uint16_t*>(base);
        const size_t q = ((size_t)rt * (n >> 5) + kb) * 1024 + lane * 8;
        return b8x2{ld8h<COH>(h, q, ok), ld8h<COH>(h, q + 512, ok)};
    } else {
        return ld4<COH>(static_cast<const float*>(base), ((size_t)rt * (n >> 4) + kb) * 256 + lane * 4, ok);
    }
}
// Store value v of element (r, c).
template <class P, bool COH>
__device__ __forceinline__ void st_tile(void* base, int r, int n, int c, float v) {
    const size_t q = tile_idx<P>(r, c, n);
    if constexpr (P::kBf16) {
        uint16_t* h = static_cast<uint16_t*>(base);
        const uint16_t hi = bf16_bits(v);
        st1h<COH>(h, q, hi);
        st1h<COH>(h, q + 512, bf16_bits(v - bf16_value(hi)));
    } else {
        st1<COH>(static_cast<float*>(base), q, v);
    }
}

// The bf16 pair copy of y_hat (the tap source) keeps one row of M values per
// latent, as n/32 blocks of [32 hi | 32 lo] (an operand's two loads share a
// 128-byte line); store value v of channel c of the row starting at `row`.
template <bool COH>
__device__ __forceinline__ void st_pair_row(uint16_t* h, size_t row, int c, float v) {
    const uint16_t hi = bf16_bits(v);
    const size_t q = row + (size_t)(c >> 5) * 64 + (c & 31);
    st1h<COH>(h, q, hi);
    st1h<COH>(h, q + 32, bf16_bits(v - bf16_value(hi)));
}

// Rows of one step: B images x n latents; row r is image r / n, grid row
// i0 + r % n, column t - lambda*i.
struct StepRows {
    int t, n, i0, nrows;
    int r0;     // grouped decode: first entry of the step's rows in StepArgs::rowlat
};

struct Row {
    bool valid;
    int b, i, j;
    size_t lat;
};

__device__ __forceinline__ Row step_row(const StepArgs& a, const StepRows& s, int r) {
    Row w;
    w.valid = r < s.nrows;
    w.b = w.i = w.j = 0;
    w.lat = 0;
    if (a.rowlat) {
        // grouped decode: the group's rows are listed
        if (w.valid) {
            const int lat = a.rowlat[s.r0 + r], hw = a.H * a.W;
            w.b = lat / hw;
            w.i = (lat - w.b * hw) / a.W;
            w.j = lat - w.b * hw - w.i * a.W;
            w.lat = (size_t)lat;
        }
        return w;
    }
    if (w.valid) {
        w.b = r / s.n;
        w.i = s.i0 + (r - w.b * s.n);
        w.j = s.t - a.lambda * w.i;
        w.lat = ((size_t)w.b * a.H + w.i) * a.W + w.j;
    }
    return w;
}

// First grid row and latent count of step t.
__host__ __device__ __forceinline__ void step_span(int H, int W, int lambda, int t, int& i0, int& n) {
    const int lo = t - (W - 1);
    i0 = lo > 0 ? (lo + lambda - 1) / lambda : 0;
    const int i1 = (H - 1) < t / lambda ? (H - 1) : t / lambda;
    n = i1 - i0 + 1;
}

__host__ __device__ __forceinline__ StepRows step_rows(int H, int W, int B, int lambda, int t) {
    StepRows s;
    s.t = t;
    step_span(H, W, lambda, t, s.i0, s.n);
    s.nrows = B * s.n;
    s.r0 = 0;
    return s;
}

// The layer-2 output of step s: h2 for even steps, h2b for odd ones (the
// dataflow driver double-buffers it by step parity; the other drivers pass
// the same array twice).
__device__ __forceinline__ void* h2_of(const StepArgs& a, const StepRows& s) { return (s.t & 1) ? a.h2b : a.h2; }

// XCD-aware job of block b: column tile ct (always on XCD ct % 8) and row
// tile rt, for kXcds * ceil(nct / kXcds) * nrt blocks.
struct Job {
    bool valid;
    int ct, rt;
};

__device__ __forceinline__ Job xcd_job(int b, int nct, int nrt) {
    const int x = b % kXcds, slot = b / kXcds;
    const int nct_x = (nct - x + kXcds - 1) / kXcds;
    Job j{false, 0, 0};
    if (nct_x <= 0) return j;
    j.rt = slot / nct_x;
    j.ct = (slot - j.rt * nct_x) * kXcds + x;
    j.valid = j.rt < nrt;
    return j;
}

__host__ __device__ __forceinline__ int xcd_blocks(int nct, int nrt) {
    return kXcds * ((nct + kXcds - 1) / kXcds) * nrt;
}

__host__ __device__ __forceinline__ int ntiles(int n) { return (n + kTile - 1) / kTile; }

// Jobs compute kC adjacent column tiles ("a column group") of one 16-row
// tile: the activation operand is loaded once for all of them.  Column
// groups of the main job of each phase (l3 keeps its own grouping: value
// group x channel tile).
template <class P>
__host__ __device__ __forceinline__ int phase_cols(const StepArgs& a, int ph) {
    switch (ph) {
        case PH_A: return a.Np1 / kTile / P::kC;
        case PH_B: return a.Np2 / kTile / P::kC;
        default: return (a.ec ? 1 : 2) * a.M / kTile;   // PH_C: value group x channel tile (ec: channel tile)
    }
}
template <class P>
__host__ __device__ __forceinline__ int phase_blocks(const StepArgs& a, const StepRows& s, int ph) {
    return xcd_blocks(phase_cols<P>(a, ph), ntiles(s.nrows));
}
// one k-part of the old-tap context of the latents of step s (nrows may be 0)
template <class P>
__host__ __device__ __forceinline__ int ctxo_blocks(const StepArgs& a, const StepRows& s) {
    if (a.n_old == 0 || s.nrows == 0) return 0;
    return xcd_blocks(2 * a.M / kTile / P::kC, ntiles(s.nrows));
}

// The work of one step: main blocks of each phase and which of the
// kParts * nc old-tap context jobs of the next step ride along with it:
// phase ph takes jobs [cut[ph], cut[ph + 1]) (part-major: job j is part
// j / nc).  A phase lasts as long as its busiest workgroup, so the context
// jobs are shared evenly among the phases as far as the slots left free in
// the last round of each phase's own jobs allow (a.slots workgroups run at
// once), then fill the remaining free slots; only what is left adds rounds,
// spread over the phases (phase A, whose own jobs are the longest, takes
// three quarters of an even share).  With fp32 the last part's jobs all run in
// the last phase, after the other parts, and add them in (see ctxo_job).
// Cuts are multiples of 8, which keeps every job on the XCD its column tile
// belongs to (nc and every phase's block count are multiples of 8).
struct StepWork {
    int nb[kMaxPhases];
    int cut[kMaxPhases + 1];
    int nc;
    // element i by selects (a runtime index into a local array would put the
    // array in scratch memory)
    __host__ __device__ __forceinline__ int blocks(int i) const {
        return i == 0 ? nb[0] : i == 1 ? nb[1] : i == 2 ? nb[2] : nb[3];
    }
    __host__ __device__ __forceinline__ int first(int i) const {
        return i == 0 ? cut[0] : i == 1 ? cut[1] : i == 2 ? cut[2] : i == 3 ? cut[3] : cut[4];
    }
};
template <class P>
__host__ __device__ __forceinline__ StepWork step_work(const StepArgs& a, const StepRows& s, const StepRows& s1) {
    // phases that share the context jobs, and the jobs they share
    constexpr int last = PH_C;
    constexpr int nph = last - P::kFirst;
    StepWork w;
    w.nc = ctxo_blocks<P>(a, s1);
    const int G = a.slots;
    int left = (P::kParts - 1) * w.nc;
    // an even share per phase first (less contention), within free slots
    const int share = ((left + nph - 1) / nph + kXcds - 1) / kXcds * kXcds;
    int take[kMaxPhases], free_slots[kMaxPhases];
#pragma unroll
    for (int ph = 0; ph < kMaxPhases; ++ph) {
        w.nb[ph] = ph < P::kFirst ? 0 : phase_blocks<P>(a, s, ph);
        const int nb = w.nb[ph];
        free_slots[ph] = ph < P::kFirst || ph >= last || nb == 0 ? 0 : ((nb + G - 1) / G * G - nb) / kXcds * kXcds;
        int t = left < share ? left : share;
        take[ph] = t < free_slots[ph] ? t : free_slots[ph];
        free_slots[ph] -= take[ph];
        left -= take[ph];
    }
#pragma unroll
    for (int ph = 0; ph < kMaxPhases; ++ph) {
        const int t = left < free_slots[ph] ? left : free_slots[ph];
        take[ph] += t;
        left -= t;
    }
    const int extra = ((left + nph - 1) / nph + kXcds - 1) / kXcds * kXcds;
    w.cut[0] = 0;
#pragma unroll
    for (int ph = 0; ph < kMaxPhases; ++ph) {
        if (ph >= P::kFirst && ph < last) {
            // layer 1's own jobs are the longest, so phase A takes three
            // quarters of an even share and the phase before C the rest
            int e = left < extra ? left : extra;
            if (ph == PH_A) e = e * 3 / 4 / kXcds * kXcds;
            if (ph == last - 1) e = left;
            take[ph] += e;
            left -= e;
        }
        if (ph == PH_C) take[ph] = w.nc;   // the last part
        w.cut[ph + 1] = w.cut[ph] + take[ph];
    }
    return w;
}

// A wave's partial sums of kC 16x16 tiles over k-blocks [kb0, kb1): w points
// at the lane's operand of k-block 0 of the first tile's packed weight column
// (tile c at w + c * ws).  The loads of up to P::kKbw k-blocks are issued
// before the MFMAs that use them (indices past the range are clamped, so every
// load is unconditional); la(kb) must be branch-free.  Each activation operand
// feeds kC independent MFMA chains.
template <class P, class LoadA>
__device__ __forceinline__ void wave_dot(const typename P::B* __restrict__ w, size_t ws, int kb0, int kb1, LoadA la,
                                         f4 (&acc)[P::kC]) {
    constexpr int kKbw = P::kKbw, C = P::kC;
    for (int kc = kb0; kc < kb1; kc += kKbw) {
        typename P::A av[kKbw];
        typename P::B bv[kKbw][C];
#pragma unroll
        for (int u = 0; u < kKbw; ++u) {
            const int k = min(kc + u, kb1 - 1);
            av[u] = la(k);
#pragma unroll
            for (int c = 0; c < C; ++c) bv[u][c] = w[c * ws + (size_t)k * 64];
        }
#pragma unroll
        for (int u = 0; u < kKbw; ++u)
            if (kc + u < kb1)
#pragma unroll
                for (int c = 0; c < C; ++c) acc[c] = P::mma(av[u], bv[u][c], acc[c]);
    }
}

// The four waves of a block split the k-blocks [klo, khi) (default: all nkb)
// of column group cg; k-blocks below `ksplit` are loaded by la_lo, the rest
// by la_hi.  Afterwards waves 0..3 hold in v[c] the full sum of tile c's row
// 4*(lane/16) + wave, column lane%16 (the other waves get 0).  red holds
// kWaves * kC rows.  Ends with a block barrier, so `red` may be reused.
template <class P, class LoadLo, class LoadHi>
__device__ __forceinline__ void block_tiles2(f4 (*red)[64], const void* __restrict__ wp, int nkb, int cg, int ksplit,
                                             LoadLo la_lo, LoadHi la_hi, float (&v)[P::kC], int klo = 0,
                                             int khi = -1) {
    constexpr int C = P::kC;
    const int wave = wave_id(), lane = threadIdx.x & 63;
    if (khi < 0) khi = nkb;
    const int per = (khi - klo + kWaves - 1) / kWaves;
    const int kb0 = min(khi, klo + wave * per), kb1 = min(khi, kb0 + per);
    const size_t ws = (size_t)nkb * 64;
    const typename P::B* w = static_cast<const typename P::B*>(wp) + (size_t)cg * C * ws + lane;
    f4 acc[C];
#pragma unroll
    for (int c = 0; c < C; ++c) acc[c] = zero4();
    wave_dot<P>(w, ws, kb0, min(kb1, ksplit), la_lo, acc);
    wave_dot<P>(w, ws, max(kb0, ksplit), kb1, la_hi, acc);
#pragma unroll
    for (int c = 0; c < C; ++c) red[wave * C + c][lane] = acc[c];
    __syncthreads();
#pragma unroll
    for (int c = 0; c < C; ++c) {
        v[c] = 0.0f;
        if (wave < 4) {
#pragma unroll
            for (int w2 = 0; w2 < kWaves; ++w2) v[c] += red[w2 * C + c][lane][wave];
        }
    }
    __syncthreads();
}

template <class P, class LoadA>
__device__ __forceinline__ void block_tiles(f4 (*red)[64], const void* __restrict__ wp, int nkb, int cg, LoadA la,
                                            float (&v)[P::kC], int klo = 0, int khi = -1) {
    block_tiles2<P>(red, wp, nkb, cg, nkb, la, la, v, klo, khi);
}

// Output column of tile c of column group cg for this lane.
template <class P>
__device__ __forceinline__ int group_col(int cg, int c) {
    return (cg * P::kC + c) * kTile + (threadIdx.x & 15);
}

// ---------------------------------------------------------------------------
// Pre-loop job b: P1[lat][n] = b_hoist[n] + sum_k psi[lat][k] * W1[n][k]
// (k < 2M), a plain dense product over all latents.  A workgroup computes a
// (32 RT)-latent x 64-column block; its four waves form a 2 x 2 grid, each
// wave RT row tiles x 2 column tiles over the whole K, so every activation
// load feeds two MFMA chains and every weight load RT, and no cross-wave
// reduction is needed.  Column blocks are placed XCD-aware.
constexpr int kHoistCols = 4;    // 16-column tiles per workgroup

template <int RT>
__host__ __device__ __forceinline__ int hoist_blocks(const StepArgs& a) {
    const int ncb = (a.Np1 / kTile + kHoistCols - 1) / kHoistCols;
    const int nrb = (a.B * a.H * a.W + kTile * 2 * RT - 1) / (kTile * 2 * RT);
    return xcd_blocks(ncb, nrb);
}

// RT row tiles per wave, KB k-blocks in flight per wave.
template <class P, bool COH, int RT, int KB>
__device__ __forceinline__ void hoist_job(const StepArgs& a, int b) {
    using A = typename P::A;
    using Bw = typename P::B;
    const int nlat = a.B * a.H * a.W;
    const int nct = a.Np1 / kTile;
    const int ncb = (nct + kHoistCols - 1) / kHoistCols;
    const Job jb = xcd_job(b, ncb, (nlat + kTile * 2 * RT - 1) / (kTile * 2 * RT));
    if (!jb.valid) return;
    const int wave = wave_id(), lane = threadIdx.x & 63, kq = lane >> 4;
    const int rt0 = jb.rt * 2 * RT + (wave >> 1) * RT;          // this wave's RT row tiles
    const int ct0 = jb.ct * kHoistCols + (wave & 1) * 2;        // and two column tiles
    const float* psi = a.cp->psi;
    const int nkb = 2 * a.M / P::kK;
    int r[RT];
    bool rv[RT], cv[2];
    const Bw* w[2];
#pragma unroll
    for (int i = 0; i < RT; ++i) {
        r[i] = (rt0 + i) * kTile + (lane & 15);
        rv[i] = r[i] < nlat;
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        cv[j] = ct0 + j < nct;                                   // wave-uniform
        w[j] = static_cast<const Bw*>(a.wp_hoist) + (size_t)(cv[j] ? ct0 + j : 0) * nkb * 64 + lane;
    }
    auto la = [&](int i, int kb) -> A {
        if constexpr (P::kBf16) {
            const size_t q = (size_t)r[i] * 2 * a.M + kb * 32 + kq * 8;
            return split8(ld4<false>(psi, q, rv[i]), ld4<false>(psi, q + 4, rv[i]));
        } else {
            return ld4<false>(psi, (size_t)r[i] * 2 * a.M + kb * kTile + kq * 4, rv[i]);
        }
    };
    f4 acc[RT][2];
#pragma unroll
    for (int i = 0; i < RT; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = zero4();
    for (int kc = 0; kc < nkb; kc += KB) {
        A av[KB][RT];
        Bw bv[KB][2];
#pragma unroll
        for (int u = 0; u < KB; ++u) {
            const int k = min(kc + u, nkb - 1);
#pragma unroll
            for (int i = 0; i < RT; ++i) av[u][i] = la(i, k);
#pragma unroll
            for (int j = 0; j < 2; ++j) bv[u][j] = w[j][(size_t)k * 64];
        }
#pragma unroll
        for (int u = 0; u < KB; ++u)
            if (kc + u < nkb)
#pragma unroll
                for (int i = 0; i < RT; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j) acc[i][j] = P::mma(av[u][i], bv[u][j], acc[i][j]);
    }
    // lane holds rows 4*(lane/16) + q of each tile, column lane%16
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        if (!cv[j]) continue;
        const int n = (ct0 + j) * kTile + (lane & 15);
        const float bias = a.b_hoist[n];
#pragma unroll
        for (int i = 0; i < RT; ++i)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int ro = (rt0 + i) * kTile + kq * 4 + q;
                if (ro < nlat) st1<COH>(a.p1, (size_t)ro * a.Np1 + n, acc[i][j][q] + bias);
            }
    }
}

// Tap gather of k-block kb of a row's taps (fp32: y_hat, bf16: its pair
// form), for the old taps (tap-major, `old` true) or the new taps.  A k-block
// never straddles two taps (M is a multiple of the k-block).
// yhat: the fp32 reconstruction (the bf16 loads read a.ybf).
template <class P, bool COH, bool R3 = true>
__device__ __forceinline__ typename P::A ld_tap_from(const StepArgs& a, const float* yhat, const Row& w, int kb,
                                                     int kq, bool old) {
    const int M = a.M;
    const int tap = kb * P::kK / M;
    const int c = kb * P::kK - tap * M + kq * (P::kK / 4);
    int dy, dx;
    if (old) {
        // the tap's row (0 = row -R) and the row's first tap, wave-uniform
        // (nested selects: a loop here costs the old-tap jobs many SGPRs)
        static_assert(kMaxRadius == 3, "rows -3..0");
        // (R3 false: masks of radius at most 2, whose old taps lie in three rows)
        const int row = tap < a.old_start[0] ? 0 : (tap < a.old_start[1] ? 1 : (!R3 || tap < a.old_start[2] ? 2 : 3));
        const int first = row == 0 ? 0 : (row == 1 ? a.old_start[0] : (!R3 || row == 2 ? a.old_start[1] : a.old_start[2]));
        dy = row - a.R;
        dx = tap - first - a.R;
    } else {
        dy = tap - 1;
        dx = tap ? -1 : a.new_dx0;
    }
    const int ii = w.i + dy, jj = w.j + dx;
    const bool ok = w.valid && ii >= 0 && jj >= 0 && jj < a.W;
    const size_t lat = ((size_t)w.b * a.H + ii) * a.W + jj;
    if constexpr (P::kBf16) {
        // c = 32 * (k-block in the latent's row) + 8 * kq
        const size_t q = lat * 2 * M + (size_t)(c >> 5) * 64 + (c & 31);
        return b8x2{ld8h<COH>(a.ybf, q, ok), ld8h<COH>(a.ybf, q + 32, ok)};
    } else {
        return ld4<COH>(yhat, lat * M + c, ok);
    }
}
template <class P, bool COH, bool R3 = true>
__device__ __forceinline__ typename P::A ld_tap(const StepArgs& a, const Row& w, int kb, int kq, bool old) {
    return ld_tap_from<P, COH, R3>(a, P::kBf16 ? nullptr : a.cp->y_hat, w, kb, kq, old);
}

// ---------------------------------------------------------------------------
// Job j of the old-tap context of the latents of step s: k-part part = j / nc
// (a contiguous range of the k-blocks of the gathered old taps, tap-major)
// of block j % nc:  ctxo[part][r][n] = sum_{k in part} taps[r][k] Wc[k][n].
// With fp32 the last part runs after the others and stores the whole sum
// (its own part plus theirs), so layer 1 reads one value per element.
template <class P, bool COH>
__device__ __forceinline__ void ctxo_tile(const StepArgs& a, const StepRows& s, int part, Job jb, f4 (*red)[64]) {
    constexpr int C = P::kC;
    const int M = a.M;
    const int wave = wave_id(), lane = threadIdx.x & 63, kq = lane >> 4;
    const int ro = wave < 4 ? jb.rt * kTile + kq * 4 + wave : s.nrows;
    const bool vo = ro < s.nrows;
    // double-buffered by step parity: jobs for step s.t may run while the
    // context of step s.t - 1 is still being read from the other half
    const size_t cpart = (size_t)a.max_rows * 2 * M;
    const int NP = a.ctx_parts;
    const size_t q = (size_t)(s.t & 1) * NP * cpart;
    float prev[C], v[C];
#pragma unroll
    for (int c = 0; c < C; ++c) {
        prev[c] = 0.0f;
        if (part == NP - 1) {
            const size_t e = q + tile_idx<PF32>(ro, group_col<P>(jb.ct, c), 2 * M);
#pragma unroll
            for (int p2 = 0; p2 < NP - 1; ++p2) prev[c] += ld1<COH>(a.ctxo, e + p2 * cpart, vo);
        }
    }
    const Row w = step_row(a, s, jb.rt * kTile + (lane & 15));
    const int nkb = a.n_old * M / P::kK;
    const int klo = nkb * part / NP, khi = nkb * (part + 1) / NP;
    if (a.R == kMaxRadius) {   // (wave-uniform)
        auto la = [&](int kb) { return ld_tap<P, COH, true>(a, w, kb, kq, true); };
        block_tiles<P>(red, a.wp_old, nkb, jb.ct, la, v, klo, khi);
    } else {
        auto la = [&](int kb) { return ld_tap<P, COH, false>(a, w, kb, kq, true); };
        block_tiles<P>(red, a.wp_old, nkb, jb.ct, la, v, klo, khi);
    }
    if (vo) {
#pragma unroll
        for (int c = 0; c < C; ++c)
            st1<COH>(a.ctxo, q + part * cpart + tile_idx<PF32>(ro, group_col<P>(jb.ct, c), 2 * M), v[c] + prev[c]);
    }
}
template <class P, bool COH>
__device__ __forceinline__ void ctxo_job(const StepArgs& a, const StepRows& s, int j, int nc, f4 (*red)[64]) {
    const int part = j / nc;
    const Job jb = xcd_job(j - part * nc, 2 * a.M / kTile / P::kC, ntiles(s.nrows));
    if (jb.valid) ctxo_tile<P, COH>(a, s, part, jb, red);
}

// Phase A, fp32: layer 1 of step s over [new taps ; old-tap context].
template <bool COH>
__device__ __forceinline__ void l1_fold_tile(const StepArgs& a, const StepRows& s, Job jb, f4 (*red)[64]) {
    constexpr int C = PF32::kC;
    const int wave = wave_id(), lane = threadIdx.x & 63, kq = lane >> 4;
    const int M = a.M;
    // epilogue operands first: the hoisted part of this wave's row
    const int ro = wave < 4 ? jb.rt * kTile + kq * 4 + wave : s.nrows;   // epilogue row of this wave
    const Row v = step_row(a, s, ro);
    float z[C], acc[C];
#pragma unroll
    for (int c = 0; c < C; ++c) z[c] = ld1<COH>(a.p1, v.lat * a.Np1 + group_col<PF32>(jb.ct, c), v.valid);
    const int r = jb.rt * kTile + (lane & 15);
    const Row w = step_row(a, s, r);
    const int knew = kMaxNew * M;
    const size_t cpart = (size_t)a.max_rows * 2 * M;
    // the old-tap context: the last part's slot holds the whole sum
    const int NP = a.ctx_parts;
    const float* ctx = a.ctxo + ((size_t)(s.t & 1) * NP + NP - 1) * cpart;
    const int kbn = knew / kTile;
    auto la_new = [&](int kb) { return ld_tap<PF32, COH>(a, w, kb, kq, false); };
    auto la_ctx = [&](int kb) -> f4 { return ld_tile<PF32, COH>(ctx, jb.rt, 2 * M, kb - kbn, w.valid); };
    block_tiles2<PF32>(red, a.wp_l1, (knew + 2 * M) / kTile, jb.ct, knew / kTile, la_new, la_ctx, acc);
    if (v.valid) {
#pragma unroll
        for (int c = 0; c < C; ++c)
            st_tile<PF32, COH>(a.h1, ro, a.Np1, group_col<PF32>(jb.ct, c), lrelu(acc[c] + z[c], a.slope));
    }
}
template <bool COH>
__device__ __forceinline__ void l1_fold_job(const StepArgs& a, const StepRows& s, int b, f4 (*red)[64]) {
    const Job jb = xcd_job(b, a.Np1 / kTile / PF32::kC, ntiles(s.nrows));
    if (jb.valid) l1_fold_tile<COH>(a, s, jb, red);
}

// Phase A, bf16: layer 1 of step s over [new taps ; old-tap context], with the
// new taps' context folded into layer 1 as for fp32: F = W1[:, 2M:] . Wc[new]
// is formed from the bf16 weights in fp64 at plan time and carried as a bf16
// pair F_hi + F_lo (panels wp_new, wp_new_lo), so the fold adds no coarse
// rounding; a new-tap k-block is hi.F_hi + lo.F_hi + hi.F_lo.  The old-tap
// context (its last k-part holds the whole sum) is carried as a pair against
// W1[:, 2M:]; the context bias is folded into P1.
template <bool COH>
__device__ __forceinline__ void l1_fold_bf16_tile(const StepArgs& a, const StepRows& s, Job jb, f4 (*red)[64]) {
    // k-blocks a wave loads before its MFMAs: all ten of a 4K step's wave in
    // one batch in the phase kernels (245 registers, still two waves per
    // SIMD); five in the persistent and dataflow kernels, whose loop state
    // would otherwise spill
    constexpr int C = PBF16::kC, KBW = COH ? 5 : 10;
    const int wave = wave_id(), lane = threadIdx.x & 63, kq = lane >> 4;
    const int M = a.M;
    // epilogue operands first: the hoisted part of this wave's row
    const int ro = wave < 4 ? jb.rt * kTile + kq * 4 + wave : s.nrows;
    const Row v = step_row(a, s, ro);
    float z[C];
#pragma unroll
    for (int c = 0; c < C; ++c) z[c] = ld1<COH>(a.p1, v.lat * a.Np1 + group_col<PBF16>(jb.ct, c), v.valid);
    const int r = jb.rt * kTile + (lane & 15);
    const Row w = step_row(a, s, r);
    const int kbn = kMaxNew * M / PBF16::kK, kbc = 2 * M / PBF16::kK, nkb = kbn + kbc;
    const int per = (nkb + kWaves - 1) / kWaves;
    const int kb0 = min(nkb, wave * per), kb1 = min(nkb, kb0 + per);
    const int NP = a.ctx_parts;
    const size_t cpart = (size_t)a.max_rows * 2 * M;
    const float* ctx = a.ctxo + ((size_t)(s.t & 1) * NP + NP - 1) * cpart;
    f4 acc[C];
#pragma unroll
    for (int c = 0; c < C; ++c) acc[c] = zero4();
    {   // new taps against the pair weights
        const b8* wh = static_cast<const b8*>(a.wp_new) + (size_t)jb.ct * C * kbn * 64 + lane;
        const b8* wl = static_cast<const b8*>(a.wp_new_lo) + (size_t)jb.ct * C * kbn * 64 + lane;
        const int e1 = min(kb1, kbn);
        for (int kc = kb0; kc < e1; kc += KBW) {
            b8x2 av[KBW];
            b8 bh[KBW][C], bl[KBW][C];
#pragma unroll
            for (int u = 0; u < KBW; ++u) {
                const int k = min(kc + u, e1 - 1);
                av[u] = ld_tap<PBF16, COH>(a, w, k, kq, false);
#pragma unroll
                for (int c = 0; c < C; ++c) {
                    bh[u][c] = wh[(size_t)(c * kbn + k) * 64];
                    bl[u][c] = wl[(size_t)(c * kbn + k) * 64];
                }
            }
#pragma unroll
            for (int u = 0; u < KBW; ++u)
                if (kc + u < e1)
#pragma unroll
                    for (int c = 0; c < C; ++c) {
                        acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[u].hi, bh[u][c], acc[c], 0, 0, 0);
                        acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[u].lo, bh[u][c], acc[c], 0, 0, 0);
                        acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[u].hi, bl[u][c], acc[c], 0, 0, 0);
                    }
        }
    }
    {   // the old-tap context: 8 values of row r, two 4-value chunks of the fp32 tile order
        const b8* w1 = static_cast<const b8*>(a.wp_l1) + (size_t)jb.ct * C * kbc * 64 + lane;
        for (int kc = max(kb0, kbn); kc < kb1; kc += KBW) {
            b8x2 av[KBW];
            b8 bv[KBW][C];
#pragma unroll
            for (int u = 0; u < KBW; ++u) {
                const int kk = min(kc + u, kb1 - 1) - kbn, c0 = kk * PBF16::kK + kq * 8;
                av[u] = split8(ld4<COH>(ctx, tile_idx<PF32>(r, c0, 2 * M), w.valid),
                               ld4<COH>(ctx, tile_idx<PF32>(r, c0 + 4, 2 * M), w.valid));
#pragma unroll
                for (int c = 0; c < C; ++c) bv[u][c] = w1[(size_t)(c * kbc + kk) * 64];
            }
#pragma unroll
            for (int u = 0; u < KBW; ++u)
                if (kc + u < kb1)
#pragma unroll
                    for (int c = 0; c < C; ++c) acc[c] = PBF16::mma(av[u], bv[u][c], acc[c]);
        }
    }
#pragma unroll
    for (int c = 0; c < C; ++c) red[wave * C + c][lane] = acc[c];
    __syncthreads();
    float o[C];
#pragma unroll
    for (int c = 0; c < C; ++c) {
        o[c] = 0.0f;
        if (wave < 4) {
#pragma unroll
            for (int w2 = 0; w2 < kWaves; ++w2) o[c] += red[w2 * C + c][lane][wave];
        }
    }
    __syncthreads();
    if (v.valid) {
#pragma unroll
        for (int c = 0; c < C; ++c)
            st_tile<PBF16, COH>(a.h1, ro, a.Np1, group_col<PBF16>(jb.ct, c), lrelu(o[c] + z[c], a.slope));
    }
}
template <bool COH>
__device__ __forceinline__ void l1_fold_bf16_job(const StepArgs& a, const StepRows& s, int b, f4 (*red)[64]) {
    const Job jb = xcd_job(b, a.Np1 / kTile / PBF16::kC, ntiles(s.nrows));
    if (jb.valid) l1_fold_bf16_tile<COH>(a, s, jb, red);
}

// Phase B: layer 2.
template <class P, bool COH>
__device__ __forceinline__ void l2_tile(const StepArgs& a, const StepRows& s, Job jb, f4 (*red)[64]) {
    constexpr int C = P::kC;
    const int wave = wave_id(), lane = threadIdx.x & 63, kq = lane >> 4;
    float bias[C], acc[C];
#pragma unroll
    for (int c = 0; c < C; ++c) bias[c] = a.b2[group_col<P>(jb.ct, c)];
    const int r = jb.rt * kTile + (lane & 15);
    const bool valid = r < s.nrows;
    auto la = [&](int kb) { return ld_tile<P, COH>(a.h1, jb.rt, a.Np1, kb, valid); };
    block_tiles<P>(red, a.wp2, a.Np1 / P::kK, jb.ct, la, acc);
    const int ro = jb.rt * kTile + kq * 4 + wave;
    if (wave < 4 && ro < s.nrows) {
#pragma unroll
        for (int c = 0; c < C; ++c)
            st_tile<P, COH>(h2_of(a, s), ro, a.Np2, group_col<P>(jb.ct, c), lrelu(acc[c] + bias[c], a.slope));
    }
}
template <class P, bool COH>
__device__ __forceinline__ void l2_job(const StepArgs& a, const StepRows& s, int b, f4 (*red)[64]) {
    const Job jb = xcd_job(b, a.Np2 / kTile / P::kC, ntiles(s.nrows));
    if (jb.valid) l2_tile<P, COH>(a, s, jb, red);
}

__device__ __forceinline__ int scale_index(const float* tab, int L, float sg) {
    // #{l in [0, L-2] : tab[l] < sg}; tab strictly increasing -> lower bound
    int lo = 0, hi = L - 1;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (tab[mid] < sg) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

template <int KC>
struct L3Smem {
    static constexpr int NT0 = KC == 1 ? 1 : 6;
    static constexpr int NT1 = KC;
    static constexpr int NTM = NT0 > NT1 ? NT0 : NT1;
    f4 red[kWaves][NTM][64];
    float tab[kMaxTable];
};

// Phase C: layer 3 and the parameter epilogue.  Job column vg * G + cg:
// channel group cg (16 channels), value group vg (0: the columns the mean
// needs -- K=1: mean, K=3: 3 logits and 3 component means; 1: the scales).
// The scale table must already be in sm.tab.
template <class P, int KC, bool COH>
__device__ __forceinline__ void l3_tile(const StepArgs& a, const StepRows& s, Job jb, L3Smem<KC>& sm) {
    using A = typename P::A;
    using Bw = typename P::B;
    constexpr int NT0 = L3Smem<KC>::NT0, NT1 = L3Smem<KC>::NT1, NTM = L3Smem<KC>::NTM;
    constexpr int KBW = KC == 1 ? P::kL3Kbw1 : P::kL3Kbw3;
    const int M = a.M, G = M / kTile;
    const int vg = jb.ct / G, cg = jb.ct - vg * G, rt = jb.rt;
    const int wave = wave_id(), lane = threadIdx.x & 63, kq = lane >> 4;

    // epilogue operands of this wave's row first
    const CallPtrs* cp = a.cp;
    const int c = cg * kTile + (lane & 15);
    const int ro = wave < 4 ? rt * kTile + kq * 4 + wave : s.nrows;   // epilogue row of this wave
    const Row v = step_row(a, s, ro);
    const size_t oq = v.lat * M + c;
    float bias[NTM];
#pragma unroll
    for (int t = 0; t < NTM; ++t) bias[t] = 0.0f;
    float sin = 0.0f;
    if (vg == 0) {
#pragma unroll
        for (int t = 0; t < NT0; ++t) bias[t] = a.b3[t * M + c];
        if (v.valid) sin = cp->encode ? cp->y[oq] : (float)cp->sym[oq];
    } else {
#pragma unroll
        for (int t = 0; t < NT1; ++t) bias[t] = a.b3[(KC == 1 ? M : (6 + t) * M) + c];
    }

    const int nkb = a.Np2 / P::kK;
    const int per = (nkb + kWaves - 1) / kWaves;
    const int kb0 = min(nkb, wave * per), kb1 = min(nkb, kb0 + per);
    const int r = rt * kTile + (lane & 15);
    const bool valid = r < s.nrows;
    const Bw* __restrict__ wv = static_cast<const Bw*>(a.wp3) + lane;
    const void* h2 = h2_of(a, s);
    const int NT = vg == 0 ? NT0 : NT1;
    int cols[NTM];
#pragma unroll
    for (int t = 0; t < NTM; ++t) cols[t] = (vg == 0 ? t : (KC == 1 ? 1 : 6 + (t < NT1 ? t : 0))) * G + cg;
    f4 acc[NTM];
#pragma unroll
    for (int t = 0; t < NTM; ++t) acc[t] = zero4();
    for (int kc = kb0; kc < kb1; kc += KBW) {
        A av[KBW];
        Bw bv[KBW][NTM];
#pragma unroll
        for (int u = 0; u < KBW; ++u) {
            const int k = min(kc + u, kb1 - 1);
            av[u] = ld_tile<P, COH>(h2, rt, a.Np2, k, valid);
#pragma unroll
            for (int t = 0; t < NTM; ++t) bv[u][t] = wv[((size_t)cols[t] * nkb + k) * 64];
        }
#pragma unroll
        for (int u = 0; u < KBW; ++u)
            if (kc + u < kb1)
#pragma unroll
                for (int t = 0; t < NTM; ++t)
                    if (t < NT) acc[t] = P::mma(av[u], bv[u][t], acc[t]);
    }
#pragma unroll
    for (int t = 0; t < NTM; ++t) sm.red[wave][t][lane] = acc[t];
    __syncthreads();
    float o[NTM];
#pragma unroll
    for (int t = 0; t < NTM; ++t) {
        o[t] = bias[t];
        if (wave < 4) {
#pragma unroll
            for (int w2 = 0; w2 < kWaves; ++w2) o[t] += sm.red[w2][t][lane][wave];
        }
    }
    __syncthreads();
    if (!v.valid) return;

    const size_t lat = v.lat;
    if (vg == 1) {
        const float t0 = sm.tab[0];
#pragma unroll
        for (int k = 0; k < KC; ++k) {
            const float sg = o[k] > t0 ? o[k] : t0;
            const size_t q = (lat * KC + k) * M + c;
            cp->scale[q] = sg;
            cp->idx[q] = scale_index(sm.tab, a.L, sg);
        }
        return;
    }
    float mu;
    if constexpr (KC == 1) {
        mu = o[0];
    } else {
        const float mx = fmaxf(o[0], fmaxf(o[1], o[2]));
        float ex[3], den = 0.0f;
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            ex[k] = expf(o[k] - mx);
            den += ex[k];
        }
        mu = 0.0f;
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            const float wk = ex[k] / den;
            const size_t q = (lat * 3 + k) * M + c;
            cp->weight[q] = wk;
            cp->cmean[q] = o[3 + k];
            mu += wk * o[3 + k];
        }
    }
    float sv;
    if (cp->encode) {
        sv = rintf(sin - mu);
        cp->sym_out[oq] = (int32_t)sv;
    } else {
        sv = sin;
    }
    cp->mean[oq] = mu;
    st1<COH>(cp->y_hat, oq, sv + mu);
    if constexpr (P::kBf16) st_pair_row<COH>(a.ybf, lat * 2 * M, c, sv + mu);
}
template <class P, int KC, bool COH>
__device__ __forceinline__ void l3_job(const StepArgs& a, const StepRows& s, int b, L3Smem<KC>& sm) {
    const Job jb = xcd_job(b, 2 * (a.M / kTile), ntiles(s.nrows));
    if (jb.valid) l3_tile<P, KC, COH>(a, s, jb, sm);
}

// ---------------------------------------------------------------------------
// Entropy decoding inside the wavefront loop (rANS; K = 1).  Each symbol is
// coded with the discretised Gaussian of its scale level, one stream per
// (image, grid row, channel) holding the row's symbols in column order, so a
// step decodes at most one symbol of every stream.  Decoder state: x in
// [2^31, 2^63); pos, end: the stream's next word and its end (the init kernel
// clamps both to the caller's buffer).  A read past the end records a stream
// error and reads zero.
__device__ __forceinline__ void ec_renorm(const CallPtrs* cp, uint64_t& x, uint32_t& pos, uint32_t end,
                                          uint32_t& wnext, bool& bad) {
    if (x < (1ull << 31)) {
        bad |= pos >= end;
        x = (x << 32) | wnext;
        pos += pos < end ? 1u : 0u;
        wnext = pos < end ? cp->bits[pos] : 0u;   // (only an escape needs it this step)
    }
}
// Decode the next symbol at scale level lvl; wnext = bits[pos] (prefetched).
__device__ __forceinline__ int32_t ec_decode(const CallPtrs* cp, int lvl, uint64_t& x, uint32_t& pos, uint32_t end,
                                             uint32_t wnext, bool& bad) {
    const int n = cp->ec_n[lvl];
    const uint32_t slot = (uint32_t)x & ((1u << kEcPrecBits) - 1u);
    // the bucket's first symbol and its interval: one load in the common case
    const uint64_t ent = cp->ec_lut[(size_t)lvl * kEcLut + (slot >> kEcLutShift)];
    int u = (int)(ent & 0xffffu);
    uint32_t c0 = (uint32_t)(ent >> 16) & 0xffffu, c1 = (uint32_t)(ent >> 32);
    if (c1 <= slot) {
        // a later symbol of the bucket: at most 15 start inside it after its first
        const uint32_t* cum = cp->ec_cum + cp->ec_base[lvl];
        for (int g = 0; g < (1 << kEcLutShift) && c1 <= slot; ++g) {
            ++u;
            c0 = c1;
            c1 = cum[u + 1];
        }
    }
    x = (uint64_t)(c1 - c0) * (x >> kEcPrecBits) + slot - c0;
    ec_renorm(cp, x, pos, end, wnext, bad);
    if (u <= 2 * n) return u - n;
    // escape: the excess in 15-bit chunks, low first, each a uniform 16-bit value
    uint64_t e = 0;
    for (int q = 0; q < 5; ++q) {
        const uint32_t ch = (uint32_t)x & 0xffffu;
        x >>= kEcPrecBits;
        ec_renorm(cp, x, pos, end, wnext, bad);
        e |= (uint64_t)(ch & 0x7fffu) << (15 * q);
        if (!(ch & 0x8000u)) {
            const int64_t mag = (int64_t)(e >> 1) + n + 1;
            return (int32_t)((e & 1u) ? -mag : mag);
        }
    }
    bad = true;
    return 0;
}

// Phase C with entropy decoding: job column cg computes the mean and the
// scale tile of channel tile cg together, so that the symbol's scale level,
// the symbol (from its stream) and y_hat = s + mean come out of one job.
template <class P, bool COH>
__device__ __forceinline__ void l3_ec_tile(const StepArgs& a, const StepRows& s, Job jb, f4 (*red)[64],
                                           const float* tab) {
    using A = typename P::A;
    using Bw = typename P::B;
    constexpr int KBW = P::kL3Kbw1;   // one batch per wave, as in l3_tile
    const int M = a.M, G = M / kTile, cg = jb.ct, rt = jb.rt;
    const int wave = wave_id(), lane = threadIdx.x & 63, kq = lane >> 4;
    const CallPtrs* cp = a.cp;
    const int c = cg * kTile + (lane & 15);
    const int ro = wave < 4 ? rt * kTile + kq * 4 + wave : s.nrows;   // epilogue row of this wave
    const Row v = step_row(a, s, ro);
    // the lane's stream: state and next word first, off the critical path
    const size_t k = ((size_t)v.b * a.H + v.i) * M + c;
    uint64_t x = 0;
    uint32_t pos = 0, end = 0, wnext = 0;
    if (v.valid) {
        x = cp->ec_x[k];
        pos = cp->ec_pos[k];
        end = cp->ec_end[k];
        wnext = pos < end ? cp->bits[pos] : 0u;
    }
    const float bias0 = a.b3[c], bias1 = a.b3[M + c];

    const int nkb = a.Np2 / P::kK;
    const int per = (nkb + kWaves - 1) / kWaves;
    const int kb0 = min(nkb, wave * per), kb1 = min(nkb, kb0 + per);
    const int r = rt * kTile + (lane & 15);
    const bool valid = r < s.nrows;
    const Bw* __restrict__ w0 = static_cast<const Bw*>(a.wp3) + (size_t)cg * nkb * 64 + lane;
    const Bw* __restrict__ w1 = static_cast<const Bw*>(a.wp3) + (size_t)(G + cg) * nkb * 64 + lane;
    const void* h2 = h2_of(a, s);
    f4 acc0 = zero4(), acc1 = zero4();
    for (int kc = kb0; kc < kb1; kc += KBW) {
        A av[KBW];
        Bw b0[KBW], b1[KBW];
#pragma unroll
        for (int u = 0; u < KBW; ++u) {
            const int kk = min(kc + u, kb1 - 1);
            av[u] = ld_tile<P, COH>(h2, rt, a.Np2, kk, valid);
            b0[u] = w0[(size_t)kk * 64];
            b1[u] = w1[(size_t)kk * 64];
        }
#pragma unroll
        for (int u = 0; u < KBW; ++u)
            if (kc + u < kb1) {
                acc0 = P::mma(av[u], b0[u], acc0);
                acc1 = P::mma(av[u], b1[u], acc1);
            }
    }
    red[wave * 2][lane] = acc0;
    red[wave * 2 + 1][lane] = acc1;
    __syncthreads();
    float mu = bias0, sr = bias1;
    if (wave < 4) {
#pragma unroll
        for (int w2 = 0; w2 < kWaves; ++w2) {
            mu += red[w2 * 2][lane][wave];
            sr += red[w2 * 2 + 1][lane][wave];
        }
    }
    __syncthreads();
    if (!v.valid) return;

    const size_t oq = v.lat * M + c;
    const float sg = sr > tab[0] ? sr : tab[0];
    const int lvl = scale_index(tab, a.L, sg);
    cp->scale[oq] = sg;
    cp->idx[oq] = lvl;
    bool bad = false;
    const int32_t sv = ec_decode(cp, lvl, x, pos, end, wnext, bad);
    cp->ec_x[k] = x;
    cp->ec_pos[k] = pos;
    if (bad) __hip_atomic_store(cp->err, kErrStream, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    cp->sym_out[oq] = sv;
    cp->mean[oq] = mu;
    const float yv = (float)sv + mu;
    st1<COH>(cp->y_hat, oq, yv);
    if constexpr (P::kBf16) st_pair_row<COH>(a.ybf, v.lat * 2 * M, c, yv);
}
template <class P, bool COH>
__device__ __forceinline__ void l3_ec_job(const StepArgs& a, const StepRows& s, int b, f4 (*red)[64],
                                          const float* tab) {
    const Job jb = xcd_job(b, a.M / kTile, ntiles(s.nrows));
    if (jb.valid) l3_ec_tile<P, COH>(a, s, jb, red, tab);
}

// ---------------------------------------------------------------------------
// Entropy decoding for the 3-component mixture model (K = 3).  A symbol is
// coded with the mixture of its channel's three Gaussians around the mixture
// mean; the frequencies are built in integer arithmetic from quantised
// parameters, so that the encoder and the decoder agree bit for bit:
//   v_k = 1 + floor(4093 w_k) (4093 w_k clamped to [0, 4093]), and what
//   is left of 4096 added to the largest v_k (the first of equals);
//   q_k = rint(16 (mu_k - mu)) clamped to +-2^14 (NaN: -2^14), the
//   component's offset in sixteenths of a symbol;
//   G_l(x): the plan's integer CDF of level l on sixteenths (2^20 scale,
//   0 at and below -X_l, 2^20 at and above X_l), l = the component's level;
//   F(s) = sum_k v_k G_{l_k}(16 s + 8 - q_k), the mixture CDF at the upper
//   edge of symbol s (2^32 = all of the mass);
//   coded symbols s_lo..s_hi, s_lo = min_k floor((q_k - X_k) / 16),
//   s_hi = max_k ceil((q_k + X_k) / 16), S = s_hi - s_lo + 1, with
//   cum(s) = (s - s_lo) + floor(F(s - 1) (2^16 - S - 1) / 2^32);
//   the last slot (2^16 - 1, frequency 1) is the escape of a symbol outside,
//   whose excess e = 2 (s_lo - 1 - s) + 1 below or 2 (s - s_hi - 1) above
//   follows in 15-bit chunks as for one Gaussian.
struct MixParam {
    uint32_t v[3];
    int q[3], l[3];
    int lo, hi;
};
// The quantised parameters of one channel (weights w, component means cm,
// mixture mean mu, levels l, all as the epilogue computed them).
__device__ __forceinline__ MixParam mix_param(const CallPtrs* cp, const float (&w)[3], const float (&cm)[3], float mu,
                                              const int (&l)[3]) {
    MixParam p;
    uint32_t sum = 0, vtop = 0;
    int top = 0;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        float wf = w[k] * 4093.0f;
        if (!(wf >= 0.0f)) wf = 0.0f;
        wf = fminf(wf, 4093.0f);
        p.v[k] = 1u + (uint32_t)floorf(wf);
        sum += p.v[k];
        if (p.v[k] > vtop) {
            vtop = p.v[k];
            top = k;
        }
        float d = rintf((cm[k] - mu) * (float)kMixFine);
        if (!(fabsf(d) <= (float)kMixQmax)) d = d > 0.0f ? (float)kMixQmax : -(float)kMixQmax;
        p.q[k] = (int)d;
        p.l[k] = l[k];
    }
#pragma unroll
    for (int k = 0; k < 3; ++k)
        if (k == top) p.v[k] += 4096u - sum;
    int lo = 0x7fffffff, hi = -0x7fffffff;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        const int X = cp->mix_X[p.l[k]];
        lo = min(lo, (p.q[k] - X) >> 4);          // floor division by 16
        hi = max(hi, -((-(p.q[k] + X)) >> 4));    // ceil
    }
    p.lo = lo;
    p.hi = hi;
    return p;
}
// F(s), in units of 2^-32 of the mass.
__device__ __forceinline__ uint64_t mix_F(const CallPtrs* cp, const MixParam& p, int s) {
    uint64_t f = 0;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        const int X = cp->mix_X[p.l[k]];
        const int x = kMixFine * s + kMixFine / 2 - p.q[k];
        const uint32_t g = x <= -X ? 0u : (x >= X ? (1u << kMixCdfBits) : cp->mix_G[cp->mix_base[p.l[k]] + x + X]);
        f += (uint64_t)p.v[k] * g;
    }
    return f;
}
__device__ __forceinline__ uint32_t mix_cum(const CallPtrs* cp, const MixParam& p, int s) {
    const uint64_t R = (1u << kEcPrecBits) - (uint64_t)(p.hi - p.lo + 1) - 1u;
    return (uint32_t)(s - p.lo) + (uint32_t)((mix_F(cp, p, s - 1) * R) >> 32);
}
// Decode the next symbol of a stream coded under the mixture p.
__device__ __forceinline__ int32_t ec_decode_mix(const CallPtrs* cp, const MixParam& p, uint64_t& x, uint32_t& pos,
                                                 uint32_t end, uint32_t wnext, bool& bad) {
    bad |= p.hi - p.lo + 1 > kMixMaxSymbols;
    const uint32_t slot = (uint32_t)x & ((1u << kEcPrecBits) - 1u);
    if (slot != (1u << kEcPrecBits) - 1u) {
        // bisection: the largest s with cum(s) <= slot (cum(s_lo) = 0)
        int lo = p.lo, hi = p.hi;
        uint32_t clo = 0;
        while (lo < hi) {
            const int mid = lo + ((hi - lo + 1) >> 1);
            const uint32_t cm = mix_cum(cp, p, mid);
            if (cm <= slot) {
                lo = mid;
                clo = cm;
            } else {
                hi = mid - 1;
            }
        }
        const uint32_t c1 = mix_cum(cp, p, lo + 1);
        x = (uint64_t)(c1 - clo) * (x >> kEcPrecBits) + slot - clo;
        ec_renorm(cp, x, pos, end, wnext, bad);
        return lo;
    }
    // escape (frequency 1), then the excess in 15-bit chunks, low first
    x >>= kEcPrecBits;
    ec_renorm(cp, x, pos, end, wnext, bad);
    uint64_t e = 0;
    for (int q = 0; q < 5; ++q) {
        const uint32_t ch = (uint32_t)x & 0xffffu;
        x >>= kEcPrecBits;
        ec_renorm(cp, x, pos, end, wnext, bad);
        e |= (uint64_t)(ch & 0x7fffu) << (15 * q);
        if (!(ch & 0x8000u)) {
            const int64_t v = (e & 1u) ? (int64_t)p.lo - 1 - (int64_t)(e >> 1) : (int64_t)p.hi + 1 + (int64_t)(e >> 1);
            bad |= v < -2147483648LL || v > 2147483647LL;
            return (int32_t)v;
        }
    }
    bad = true;
    return 0;
}

// Phase C with entropy decoding, K = 3: job column cg computes all nine
// column tiles of channel tile cg (3 logits, 3 component means, 3 scales),
// so that a lane holds its channel's whole mixture, decodes the symbol from
// its stream and writes y_hat = s + mean in the same job.
template <class P, bool COH>
__device__ __forceinline__ void l3_ec3_tile(const StepArgs& a, const StepRows& s, Job jb, L3Smem<3>& sm) {
    using A = typename P::A;
    using Bw = typename P::B;
    constexpr int KBW = 2;   // k-blocks a wave loads before its MFMAs (nine weight operands each)
    constexpr int NT = 9;
    const int M = a.M, G = M / kTile, cg = jb.ct, rt = jb.rt;
    const int wave = wave_id(), lane = threadIdx.x & 63, kq = lane >> 4;
    const CallPtrs* cp = a.cp;
    const int c = cg * kTile + (lane & 15);
    const int ro = wave < 4 ? rt * kTile + kq * 4 + wave : s.nrows;   // epilogue row of this wave
    const Row v = step_row(a, s, ro);
    const size_t k = ((size_t)v.b * a.H + v.i) * M + c;
    uint64_t x = 0;
    uint32_t pos = 0, end = 0, wnext = 0;
    if (v.valid) {
        x = cp->ec_x[k];
        pos = cp->ec_pos[k];
        end = cp->ec_end[k];
        wnext = pos < end ? cp->bits[pos] : 0u;
    }
    float bias[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) bias[t] = a.b3[t * M + c];

    const int nkb = a.Np2 / P::kK;
    const int per = (nkb + kWaves - 1) / kWaves;
    const int kb0 = min(nkb, wave * per), kb1 = min(nkb, kb0 + per);
    const int r = rt * kTile + (lane & 15);
    const bool valid = r < s.nrows;
    const Bw* __restrict__ wv = static_cast<const Bw*>(a.wp3) + lane;
    const void* h2 = h2_of(a, s);
    f4 acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = zero4();
    for (int kc = kb0; kc < kb1; kc += KBW) {
        A av[KBW];
        Bw bv[KBW][NT];
#pragma unroll
        for (int u = 0; u < KBW; ++u) {
            const int kk = min(kc + u, kb1 - 1);
            av[u] = ld_tile<P, COH>(h2, rt, a.Np2, kk, valid);
#pragma unroll
            for (int t = 0; t < NT; ++t) bv[u][t] = wv[((size_t)(t * G + cg) * nkb + kk) * 64];
        }
#pragma unroll
        for (int u = 0; u < KBW; ++u)
            if (kc + u < kb1)
#pragma unroll
                for (int t = 0; t < NT; ++t) acc[t] = P::mma(av[u], bv[u][t], acc[t]);
    }
    // the nine tiles' wave sums in two rounds through the six-tile buffer
    float o[NT];
#pragma unroll
    for (int rnd = 0; rnd < 2; ++rnd) {
        const int t0 = rnd * 6, nt = rnd ? NT - 6 : 6;
#pragma unroll
        for (int t = 0; t < 6; ++t)
            if (t < nt) sm.red[wave][t][lane] = acc[t0 + t];
        __syncthreads();
#pragma unroll
        for (int t = 0; t < 6; ++t)
            if (t < nt) {
                o[t0 + t] = bias[t0 + t];
                if (wave < 4) {
#pragma unroll
                    for (int w2 = 0; w2 < kWaves; ++w2) o[t0 + t] += sm.red[w2][t][lane][wave];
                }
            }
        __syncthreads();
    }
    if (!v.valid) return;

    const size_t lat = v.lat, oq = lat * M + c;
    const float mx = fmaxf(o[0], fmaxf(o[1], o[2]));
    float ex[3], den = 0.0f;
#pragma unroll
    for (int kk = 0; kk < 3; ++kk) {
        ex[kk] = expf(o[kk] - mx);
        den += ex[kk];
    }
    float w3[3], m3[3], mu = 0.0f;
    int l3[3];
    const float t0 = sm.tab[0];
#pragma unroll
    for (int kk = 0; kk < 3; ++kk) {
        w3[kk] = ex[kk] / den;
        m3[kk] = o[3 + kk];
        mu += w3[kk] * m3[kk];
        const float sg = o[6 + kk] > t0 ? o[6 + kk] : t0;
        l3[kk] = scale_index(sm.tab, a.L, sg);
        const size_t q = (lat * 3 + kk) * M + c;
        cp->weight[q] = w3[kk];
        cp->cmean[q] = m3[kk];
        cp->scale[q] = sg;
        cp->idx[q] = l3[kk];
    }
    bool bad = false;
    const MixParam mp = mix_param(cp, w3, m3, mu, l3);
    const int32_t sv = ec_decode_mix(cp, mp, x, pos, end, wnext, bad);
    cp->ec_x[k] = x;
    cp->ec_pos[k] = pos;
    if (bad) __hip_atomic_store(cp->err, kErrStream, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    cp->sym_out[oq] = sv;
    cp->mean[oq] = mu;
    const float yv = (float)sv + mu;
    st1<COH>(cp->y_hat, oq, yv);
    if constexpr (P::kBf16) st_pair_row<COH>(a.ybf, lat * 2 * M, c, yv);
}
template <class P, bool COH>
__device__ __forceinline__ void l3_ec3_job(const StepArgs& a, const StepRows& s, int b, L3Smem<3>& sm) {
    const Job jb = xcd_job(b, a.M / kTile, ntiles(s.nrows));
    if (jb.valid) l3_ec3_tile<P, COH>(a, s, jb, sm);
}

// ---------------------------------------------------------------------------
// Context approximation (Sec. III-D): a step is a group of N wavefronts.  A
// tap of the latent's own group is not decoded yet and is replaced, channel by
// channel, by the mean of the latent's decoded in-image taps (zero when none
// is decoded); out-of-grid taps are zero.  Tap k of the mask (raster order).
__device__ __forceinline__ void mask_tap(const StepArgs& a, int k, int& dy, int& dx) {
    const int rw = a.row_w, up = a.R * rw;
    if (k < up) {
        const int q = k / rw;
        dy = q - a.R;
        dx = k - q * rw - a.R;
    } else {
        dy = 0;
        dx = k - up - a.R;
    }
}

// Job of the grouped context: k-part `part` of ctx[r][n] = sum over taps and
// channels of W_c[n][c][tap] x_tap[r][c] for one row tile and column group.
// The k order of the packed weights is channel-chunk-major (chunk q of kK
// channels, then the taps), and wave w of part p takes chunk 4p + w: it loads
// that chunk of every tap, so the fill mean of its channels is formed in
// registers from the same loads.  The parts are summed by layer 1.  NT bounds
// the mask's tap count (the taps stay in registers).
template <class P, int NT, bool COH>
__device__ __forceinline__ void gctx_tile(const StepArgs& a, const StepRows& s, int part, Job jb, f4 (*red)[64]) {
    constexpr int C = P::kC, KB = P::kK, CPL = KB / 4;   // channels per lane of a chunk
    const int wave = wave_id(), lane = threadIdx.x & 63, kq = lane >> 4;
    const int M = a.M, Q = M / KB, nt = a.n_old + kMaxNew;
    const int q = part * kWaves + wave;                  // this wave's channel chunk
    const Row w = step_row(a, s, jb.rt * kTile + (lane & 15));
    const int g = (a.lambda * w.i + w.j) / a.group;
    f4 acc[C];
#pragma unroll
    for (int c = 0; c < C; ++c) acc[c] = zero4();
    if (q < Q) {
        typename P::A x[NT];
        float sum[CPL];
#pragma unroll
        for (int e = 0; e < CPL; ++e) sum[e] = 0.0f;
        unsigned long long status = 0;                   // 2 bits per tap: 0 out, 1 decoded, 2 filled
        int known = 0;
        const int c0 = q * KB + kq * CPL;
#pragma unroll
        for (int k = 0; k < NT; ++k) {
            // (every index below is a compile-time constant, so x[] stays in registers)
            int dy, dx;
            mask_tap(a, k, dy, dx);
            const int ii = w.i + dy, jj = w.j + dx;
            const bool in = k < nt && w.valid && ii >= 0 && jj >= 0 && jj < a.W;
            const bool dec = in && (a.lambda * ii + jj) / a.group < g;
            status |= (unsigned long long)(in ? (dec ? 1u : 2u) : 0u) << (2 * k);
            known += dec;
            const size_t lat = ((size_t)w.b * a.H + ii) * a.W + jj;
            if constexpr (P::kBf16) {
                const size_t o = lat * 2 * M + (size_t)(c0 >> 5) * 64 + (c0 & 31);
                x[k] = b8x2{ld8h<COH>(a.ybf, o, dec), ld8h<COH>(a.ybf, o + 32, dec)};
            } else {
                x[k] = ld4<COH>(a.cp->y_hat, lat * M + c0, dec);
            }
        }
#pragma unroll
        for (int k = 0; k < NT; ++k) {
            if constexpr (P::kBf16) {
#pragma unroll
                for (int e = 0; e < 8; ++e) sum[e] += (float)x[k].hi[e] + (float)x[k].lo[e];
            } else {
                sum[0] += x[k].x; sum[1] += x[k].y; sum[2] += x[k].z; sum[3] += x[k].w;
            }
        }
        float mean[CPL];
#pragma unroll
        for (int e = 0; e < CPL; ++e) mean[e] = known > 0 ? sum[e] / (float)known : 0.0f;
        typename P::A fillv;
        if constexpr (P::kBf16) fillv = split8(f4{mean[0], mean[1], mean[2], mean[3]}, f4{mean[4], mean[5], mean[6], mean[7]});
        else fillv = f4{mean[0], mean[1], mean[2], mean[3]};
        const size_t ws = (size_t)nt * Q * 64;           // one column tile of the packed panel
        const typename P::B* wp = static_cast<const typename P::B*>(a.wp_all) + (size_t)jb.ct * C * ws + lane;
#pragma unroll
        for (int k = 0; k < NT; ++k) {
            if (k >= nt) continue;                       // wave-uniform
            const unsigned st = (unsigned)(status >> (2 * k)) & 3u;
            typename P::A v = x[k];
            if (st == 2u) v = fillv;                     // decoded taps and zeros (out of grid) as loaded
#pragma unroll
            for (int c = 0; c < C; ++c) acc[c] = P::mma(v, wp[c * ws + (size_t)(q * nt + k) * 64], acc[c]);
        }
    }
#pragma unroll
    for (int c = 0; c < C; ++c) red[wave * C + c][lane] = acc[c];
    __syncthreads();
    const int ro = wave < 4 ? jb.rt * kTile + kq * 4 + wave : s.nrows;
    float v[C];
#pragma unroll
    for (int c = 0; c < C; ++c) {
        v[c] = 0.0f;
        if (wave < 4) {
#pragma unroll
            for (int w2 = 0; w2 < kWaves; ++w2) v[c] += red[w2 * C + c][lane][wave];
        }
    }
    __syncthreads();
    if (ro < s.nrows) {
        const size_t cpart = (size_t)a.max_rows * 2 * M;
        const size_t base = ((size_t)(s.t & 1) * a.gparts + part) * cpart;
#pragma unroll
        for (int c = 0; c < C; ++c) st1<COH>(a.ctxo, base + tile_idx<PF32>(ro, group_col<P>(jb.ct, c), 2 * M), v[c]);
    }
}
template <class P, int NT, bool COH>
__device__ __forceinline__ void gctx_job(const StepArgs& a, const StepRows& s, int j, int nc, f4 (*red)[64]) {
    const int part = j / nc;
    const Job jb = xcd_job(j - part * nc, 2 * a.M / kTile / P::kC, ntiles(s.nrows));
    if (jb.valid) gctx_tile<P, NT, COH>(a, s, part, jb, red);
}

// Grouped decode, layer 1 over the context (the sum of the gctx parts):
// h1 = lrelu(P1 + W1[:, 2M:] . ctx), the context bias folded into P1 (fp32:
// the weights are the second block of the layer-1 panel; bf16: the context is
// carried as a pair).
template <class P, bool COH>
__device__ __forceinline__ void l1_group_tile(const StepArgs& a, const StepRows& s, Job jb, f4 (*red)[64]) {
    constexpr int C = P::kC;
    const int wave = wave_id(), lane = threadIdx.x & 63, kq = lane >> 4;
    const int M = a.M;
    const int ro = wave < 4 ? jb.rt * kTile + kq * 4 + wave : s.nrows;
    const Row v = step_row(a, s, ro);
    float z[C], acc[C];
#pragma unroll
    for (int c = 0; c < C; ++c) z[c] = ld1<COH>(a.p1, v.lat * a.Np1 + group_col<P>(jb.ct, c), v.valid);
    const int r = jb.rt * kTile + (lane & 15);
    const bool valid = r < s.nrows;
    const size_t cpart = (size_t)a.max_rows * 2 * M;
    const float* ctx = a.ctxo + (size_t)(s.t & 1) * a.gparts * cpart;
    const int np = a.gparts;
    if constexpr (P::kBf16) {
        // 8 context values of row r: two 4-value chunks of the fp32 tile order
        auto la = [&](int kb) -> b8x2 {
            const int c0 = kb * 32 + kq * 8;
            const size_t i0 = tile_idx<PF32>(r, c0, 2 * M), i1 = tile_idx<PF32>(r, c0 + 4, 2 * M);
            f4 u = zero4(), t = zero4();
            for (int p2 = 0; p2 < np; ++p2) {
                u += ld4<COH>(ctx, i0 + p2 * cpart, valid);
                t += ld4<COH>(ctx, i1 + p2 * cpart, valid);
            }
            return split8(u, t);
        };
        block_tiles<PBF16>(red, a.wp_l1, 2 * M / PBF16::kK, jb.ct, la, acc);
    } else {
        const int kbn = kMaxNew * M / kTile;             // the panel's first block (folded taps) is skipped
        auto la = [&](int kb) -> f4 {
            f4 u = zero4();
            for (int p2 = 0; p2 < np; ++p2) u += ld_tile<PF32, COH>(ctx + p2 * cpart, jb.rt, 2 * M, kb - kbn, valid);
            return u;
        };
        block_tiles<PF32>(red, a.wp_l1, (kMaxNew * M + 2 * M) / kTile, jb.ct, la, acc, kbn);
    }
    if (v.valid) {
#pragma unroll
        for (int c = 0; c < C; ++c)
            st_tile<P, COH>(a.h1, ro, a.Np1, group_col<P>(jb.ct, c), lrelu(acc[c] + z[c], a.slope));
    }
}

// The main job of phase ph (sm.tab must hold the scale table for PH_C); EC:
// phase C decodes the symbols from their rANS streams (a.ec set).
template <class P, int KC, bool COH, bool EC = false>
__device__ __forceinline__ void phase_job(int ph, const StepArgs& a, const StepRows& s, int b, f4 (*red)[64],
                                          L3Smem<KC>& sm) {
    if (ph == PH_GA) {
        const Job jb = xcd_job(b, a.Np1 / kTile / P::kC, ntiles(s.nrows));
        if (jb.valid) l1_group_tile<P, COH>(a, s, jb, red);
        return;
    }
    if constexpr (EC && KC == 1) {
        if (ph == PH_C) {
            l3_ec_job<P, COH>(a, s, b, red, sm.tab);
            return;
        }
    }
    if constexpr (EC && KC == 3) {
        if (ph == PH_C) {
            l3_ec3_job<P, COH>(a, s, b, sm);
            return;
        }
    }
    if constexpr (P::kBf16) {
        if (ph == PH_A) l1_fold_bf16_job<COH>(a, s, b, red);
        else if (ph == PH_B) l2_job<P, COH>(a, s, b, red);
        else l3_job<P, KC, COH>(a, s, b, sm);
    } else {
        if (ph == PH_A) l1_fold_job<COH>(a, s, b, red);
        else if (ph == PH_B) l2_job<P, COH>(a, s, b, red);
        else l3_job<P, KC, COH>(a, s, b, sm);
    }
}

}  // namespace wf
