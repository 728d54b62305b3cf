// Device code shared by the per-step kernels and the persistent kernel: the
// MFMA tile engine and the work of the three phases of a wavefront step.
//
// For step t (Sec. III-C):
//   phase A  h1 = lrelu(P1 + sum of pushed old-tap slots + F_new . new taps)
//            and the push of step t-1: every latent of step t-1 adds
//            F_o . y_hat into slot o of each later latent that has it as old
//            tap o
//   phase B  h2 = lrelu(W2 . h1 + b2)
//   phase C  o  = W3 . h2 + b3  -> mean / scale / index, y_hat = s + mean
// with P1 = b1 + W1[:, 2M:] . bc + W1[:, :2M] . psi hoisted before the loop
// and F = W1[:, 2M:] . Wc[tap] the per-tap folded weights.
//
// Every product runs on fp32 MFMA (v_mfma_f32_16x16x4f32).  Each wave issues
// all operand loads of its k-range before its first MFMA, and the epilogue
// operands are fetched before the products.  Jobs are placed XCD-aware:
// block b runs on XCD b % 8, and each column tile of a weight matrix is always
// computed on the same XCD, which then streams only its slice of the weights.
//
// COH selects how data produced by other workgroups of the same launch is
// accessed: with COH the activations, the reconstruction and the pushed slots
// are written and read with agent-coherent (sc1) buffer operations, so the
// persistent kernel needs no cache flush between its phases.
#pragma once

#include "wf_internal.h"

namespace wf {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kKbw = 20;   // k-blocks (16 values of k) loaded by a wave before its MFMAs
constexpr int kSc1 = 16;   // cache-policy bits of an agent-coherent buffer access

__device__ __forceinline__ f4 mfma_k16(f4 a, f4 b, f4 acc) {
    // Lane l supplies A[l%16][4*(l/16)+q] and B[4*(l/16)+q][l%16] for the q-th
    // instruction: the four instructions together sum over 16 values of k.
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, b.x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, b.y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, b.z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, b.w, acc, 0, 0, 0);
    return acc;
}

__device__ __forceinline__ float lrelu(float v, float s) { return v >= 0.0f ? v : s * v; }

__device__ __forceinline__ f4 zero4() { return f4{0.0f, 0.0f, 0.0f, 0.0f}; }

// Raw buffer resource over [p, p + 2 GiB): out-of-range accesses return zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, 0x7fffffff, 0x00020000);
}

// Loads/stores of data written by other workgroups of the same launch.
// (the buffer builtins move raw 32-bit words: bit casts, not conversions)
typedef unsigned u4 __attribute__((ext_vector_type(4)));
template <bool COH>
__device__ __forceinline__ f4 ld4(const float* base, size_t idx) {
    if (COH)
        return __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(rsrc(base), (int)(idx * 4), 0, kSc1));
    return *reinterpret_cast<const f4*>(base + idx);
}
template <bool COH>
__device__ __forceinline__ float ld1(const float* base, size_t idx) {
    if (COH)
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc(base), (int)(idx * 4), 0, kSc1));
    return base[idx];
}
template <bool COH>
__device__ __forceinline__ void st1(float* base, size_t idx, float v) {
    if (COH)
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), rsrc(base), (int)(idx * 4), 0, kSc1);
    else
        base[idx] = v;
}

// Rows of one step: B images x n latents; row r is image r / n, grid row
// i0 + r % n, column t - lambda*i.
struct StepRows {
    int t, n, i0, nrows;
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
    return s;
}

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

// Block counts of the three phases of a step.
__host__ __device__ __forceinline__ int phase_a_l1_blocks(const StepArgs& a, const StepRows& s) {
    return xcd_blocks(a.Np1 / kTile, ntiles(s.nrows));
}
__host__ __device__ __forceinline__ int phase_a_push_blocks(const StepArgs& a, const StepRows& sp, int T) {
    // the push of step sp.t is needed when a consumer step sp.t + 2 exists
    if (a.n_old == 0 || sp.nrows == 0 || sp.t + 2 >= T) return 0;
    return xcd_blocks((a.n_old * a.Np1 / kTile + kWaves - 1) / kWaves, ntiles(sp.nrows));
}
__host__ __device__ __forceinline__ int phase_b_blocks(const StepArgs& a, const StepRows& s) {
    return xcd_blocks(a.Np2 / kTile, ntiles(s.nrows));
}
__host__ __device__ __forceinline__ int phase_c_blocks(const StepArgs& a, const StepRows& s) {
    return xcd_blocks(2 * a.M / kTile, ntiles(s.nrows));
}

// A wave's partial 16x16 tile over k-blocks [kb0, kb1): w points at the
// lane's operand of k-block 0 of the tile's packed weight column; all loads
// of up to kKbw k-blocks are issued before the MFMAs that use them.
template <class LoadA>
__device__ __forceinline__ f4 wave_dot(const f4* __restrict__ w, int kb0, int kb1, LoadA la) {
    f4 acc = zero4();
    for (int kc = kb0; kc < kb1; kc += kKbw) {
        f4 av[kKbw], bv[kKbw];
#pragma unroll
        for (int u = 0; u < kKbw; ++u) {
            const int k = kc + u;
            if (k < kb1) {
                av[u] = la(k);
                bv[u] = w[(size_t)k * 64];
            }
        }
#pragma unroll
        for (int u = 0; u < kKbw; ++u)
            if (kc + u < kb1) acc = mfma_k16(av[u], bv[u], acc);
    }
    return acc;
}

// The four waves of a block split the k-blocks of one tile; afterwards every
// wave holds the full sum of tile row 4*(lane/16) + wave, column lane%16.
// Ends with a block barrier, so `red` may be reused right away.
template <class LoadA>
__device__ __forceinline__ float block_tile(f4 (*red)[64], const float* __restrict__ wp, int nkb, int ct,
                                            LoadA la) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int per = (nkb + kWaves - 1) / kWaves;
    const int kb0 = min(nkb, wave * per), kb1 = min(nkb, kb0 + per);
    const f4* w = reinterpret_cast<const f4*>(wp) + (size_t)ct * nkb * 64 + lane;
    red[wave][lane] = wave_dot(w, kb0, kb1, la);
    __syncthreads();
    const float v = red[0][lane][wave] + red[1][lane][wave] + red[2][lane][wave] + red[3][lane][wave];
    __syncthreads();
    return v;
}

// ---------------------------------------------------------------------------
// Phase A, push part: producer step sp, one wave per column tile of the
// old-tap weights (four consecutive tiles per block).
template <bool COH>
__device__ __forceinline__ void push_job(const StepArgs& a, const StepRows& sp, int b) {
    const int nct = a.n_old * a.Np1 / kTile;
    const Job jb = xcd_job(b, (nct + kWaves - 1) / kWaves, ntiles(sp.nrows));
    if (!jb.valid) return;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, kq = lane >> 4;
    const int ct = jb.ct * kWaves + wave;
    if (ct >= nct) return;
    const int M = a.M;
    const Row w = step_row(a, sp, jb.rt * kTile + (lane & 15));
    const float* yh = a.cp->y_hat;
    const size_t ybase = w.lat * M + kq * 4;
    auto la = [&](int kb) -> f4 { return w.valid ? ld4<COH>(yh, ybase + kb * kTile) : zero4(); };
    const f4* wv = reinterpret_cast<const f4*>(a.wp_old) + (size_t)ct * (M / kTile) * 64 + lane;
    const f4 acc = wave_dot(wv, 0, M / kTile, la);
    const int col = ct * kTile + (lane & 15);
    const int o = col / a.Np1, n = col - o * a.Np1;
    const int dy = a.old_dy[o], dx = a.old_dx[o], tc = sp.t + a.old_delta[o];
    int ci0, cn;
    step_span(a.H, a.W, a.lambda, tc, ci0, cn);
    const size_t ring = (size_t)(tc % a.nring) * a.max_rows;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const Row v = step_row(a, sp, jb.rt * kTile + kq * 4 + q);
        if (!v.valid) continue;
        const int ic = v.i - dy, jc = v.j - dx;   // the consumer
        if (ic >= a.H || jc < 0 || jc >= a.W) continue;
        const size_t rc = (size_t)v.b * cn + (ic - ci0);
        st1<COH>(a.slots, ((ring + rc) * a.n_old + o) * a.Np1 + n, acc[q]);
    }
}

// Phase A, layer-1 part: block b of the layer-1 jobs of step s.
template <bool COH>
__device__ __forceinline__ void l1_job(const StepArgs& a, const StepRows& s, int b, f4 (*red)[64]) {
    const Job jb = xcd_job(b, a.Np1 / kTile, ntiles(s.nrows));
    if (!jb.valid) return;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, kq = lane >> 4;
    const int M = a.M;
    // epilogue operands first: hoisted part and pushed slots of this wave's row
    const int n = jb.ct * kTile + (lane & 15);
    const int ro = jb.rt * kTile + kq * 4 + wave;
    const Row v = step_row(a, s, ro);
    float z = 0.0f;
    if (v.valid) {
        z = a.p1[v.lat * a.Np1 + n];
        const size_t sl = (((size_t)(s.t % a.nring) * a.max_rows + ro) * a.n_old) * a.Np1 + n;
        for (int o = 0; o < a.n_old; ++o) {
            const int ii = v.i + a.old_dy[o], jj = v.j + a.old_dx[o];
            if (ii >= 0 && jj >= 0 && jj < a.W) z += ld1<COH>(a.slots, sl + (size_t)o * a.Np1);
        }
    }
    const Row w = step_row(a, s, jb.rt * kTile + (lane & 15));
    const float* yh = a.cp->y_hat;
    auto la = [&](int kb) -> f4 {
        const int k0 = kb * kTile + kq * 4;
        const int tap = k0 >= M ? 1 : 0, c = k0 - tap * M;
        const int ii = w.i + a.new_dy[tap], jj = w.j + a.new_dx[tap];
        if (!w.valid || ii < 0 || jj < 0 || jj >= a.W) return zero4();
        return ld4<COH>(yh, (((size_t)w.b * a.H + ii) * a.W + jj) * M + c);
    };
    const float acc = block_tile(red, a.wp_new, a.n_new * M / kTile, jb.ct, la);
    if (v.valid) st1<COH>(a.h1, (size_t)ro * a.Np1 + n, lrelu(acc + z, a.slope));
}

// Phase B: layer 2.
template <bool COH>
__device__ __forceinline__ void l2_job(const StepArgs& a, const StepRows& s, int b, f4 (*red)[64]) {
    const Job jb = xcd_job(b, a.Np2 / kTile, ntiles(s.nrows));
    if (!jb.valid) return;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, kq = lane >> 4;
    const int n = jb.ct * kTile + (lane & 15);
    const float bias = a.b2[n];
    const int r = jb.rt * kTile + (lane & 15);
    const bool valid = r < s.nrows;
    const size_t base = (size_t)r * a.Np1 + kq * 4;
    auto la = [&](int kb) -> f4 { return valid ? ld4<COH>(a.h1, base + kb * kTile) : zero4(); };
    const float acc = block_tile(red, a.wp2, a.Np1 / kTile, jb.ct, la);
    const int ro = jb.rt * kTile + kq * 4 + wave;
    if (ro < s.nrows) st1<COH>(a.h2, (size_t)ro * a.Np2 + n, lrelu(acc + bias, a.slope));
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
template <int KC, bool COH>
__device__ __forceinline__ void l3_job(const StepArgs& a, const StepRows& s, int b, L3Smem<KC>& sm) {
    constexpr int NT0 = L3Smem<KC>::NT0, NT1 = L3Smem<KC>::NT1, NTM = L3Smem<KC>::NTM;
    constexpr int KBW = KC == 1 ? 16 : 4;
    const int M = a.M, G = M / kTile;
    const Job jb = xcd_job(b, 2 * G, ntiles(s.nrows));
    if (!jb.valid) return;
    const int vg = jb.ct / G, cg = jb.ct - vg * G, rt = jb.rt;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, kq = lane >> 4;

    // epilogue operands of this wave's row first
    const CallPtrs* cp = a.cp;
    const int c = cg * kTile + (lane & 15);
    const int ro = rt * kTile + kq * 4 + wave;
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

    const int nkb = a.Np2 / kTile;
    const int per = (nkb + kWaves - 1) / kWaves;
    const int kb0 = min(nkb, wave * per), kb1 = min(nkb, kb0 + per);
    const int r = rt * kTile + (lane & 15);
    const bool valid = r < s.nrows;
    const size_t hbase = (size_t)r * a.Np2 + kq * 4;
    const f4* __restrict__ wv = reinterpret_cast<const f4*>(a.wp3) + lane;
    const int NT = vg == 0 ? NT0 : NT1;
    int cols[NTM];
#pragma unroll
    for (int t = 0; t < NTM; ++t) cols[t] = (vg == 0 ? t : (KC == 1 ? 1 : 6 + t)) * G + cg;
    f4 acc[NTM];
#pragma unroll
    for (int t = 0; t < NTM; ++t) acc[t] = zero4();
    for (int kc = kb0; kc < kb1; kc += KBW) {
        f4 av[KBW], bv[KBW][NTM];
#pragma unroll
        for (int u = 0; u < KBW; ++u) {
            const int k = kc + u;
            if (k < kb1) {
                av[u] = valid ? ld4<COH>(a.h2, hbase + k * kTile) : zero4();
#pragma unroll
                for (int t = 0; t < NTM; ++t)
                    if (t < NT) bv[u][t] = wv[((size_t)cols[t] * nkb + k) * 64];
            }
        }
#pragma unroll
        for (int u = 0; u < KBW; ++u)
            if (kc + u < kb1)
#pragma unroll
                for (int t = 0; t < NTM; ++t)
                    if (t < NT) acc[t] = mfma_k16(av[u], bv[u][t], acc[t]);
    }
#pragma unroll
    for (int t = 0; t < NTM; ++t) sm.red[wave][t][lane] = acc[t];
    __syncthreads();
    float o[NTM];
#pragma unroll
    for (int t = 0; t < NTM; ++t)
        o[t] = sm.red[0][t][lane][wave] + sm.red[1][t][lane][wave] + sm.red[2][t][lane][wave] +
               sm.red[3][t][lane][wave] + bias[t];
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
    if (KC == 1) {
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
}

}  // namespace wf
