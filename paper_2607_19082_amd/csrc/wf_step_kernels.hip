// Per-step kernels of the wavefront decode/encode and the stream driver.
//
// One wavefront step (Sec. III-C) is four batched products and an epilogue:
//   ctx = taps . Wc            (masked 5x5 conv over the gathered causal taps)
//   h1  = [psi ; ctx + bc] . W1
//   h2  = lrelu(h1 + b1) . W2
//   o   = lrelu(h2 + b2) . W3
//   epilogue: mean/scale/index from o + b3, then y_hat = s + mean.
// Each product runs on fp32 MFMA (v_mfma_f32_16x16x4f32), one wave per 16x16
// output tile and k-slice, with the slices summed by fp32 atomics into a raw
// buffer.  The consumer adds the bias and applies the activation when it loads
// its operand, and the epilogue clears the raw buffers for the next step.
#include "wf_internal.h"

namespace wf {

typedef float f4 __attribute__((ext_vector_type(4)));

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

template <int SRC>
__global__ __launch_bounds__(64) void k_step_gemm(StepRows s, GemmArgs g) {
    const int lane = threadIdx.x;
    const int ct = blockIdx.x, rt = blockIdx.y;
    const int kb0 = blockIdx.z * g.kb_per_split;
    const int kb1 = min(g.nkb, kb0 + g.kb_per_split);
    if (kb0 >= kb1) return;

    const int kq = lane >> 4;
    const int r = rt * kTile + (lane & 15);
    const bool valid = r < s.nrows;
    int b = 0, i = 0, j = 0;
    size_t lat = 0;
    if (valid) {
        b = r / s.n;
        const int pos = g.order[s.ptr + (r - b * s.n)];
        i = pos / g.W;
        j = pos - i * g.W;
        lat = (size_t)b * g.H * g.W + pos;
    }
    const int cpb = g.M / kTile;  // k-blocks per tap
    const f4* wp = reinterpret_cast<const f4*>(g.wp) + (size_t)ct * g.nkb * 64 + lane;

    f4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int kb = kb0; kb < kb1; ++kb) {
        f4 a = {0.0f, 0.0f, 0.0f, 0.0f};
        const int k0 = kb * kTile + kq * 4;
        if (valid) {
            if (SRC == A_TAPS) {
                const int tap = kb / cpb;
                const int c = k0 - tap * g.M;
                const int ii = i + g.dy[tap], jj = j + g.dx[tap];
                if (ii >= 0 && jj >= 0 && jj < g.W)
                    a = *reinterpret_cast<const f4*>(g.y_hat + (((size_t)b * g.H + ii) * g.W + jj) * g.M + c);
            } else if (SRC == A_PSI_CTX) {
                if (k0 < 2 * g.M) {
                    a = *reinterpret_cast<const f4*>(g.psi + lat * 2 * g.M + k0);
                } else {
                    const int kc = k0 - 2 * g.M;
                    a = *reinterpret_cast<const f4*>(g.in + (size_t)r * g.ldi + kc) +
                        *reinterpret_cast<const f4*>(g.in_bias + kc);
                }
            } else {
                f4 v = *reinterpret_cast<const f4*>(g.in + (size_t)r * g.ldi + k0) +
                       *reinterpret_cast<const f4*>(g.in_bias + k0);
                a.x = lrelu(v.x, g.slope);
                a.y = lrelu(v.y, g.slope);
                a.z = lrelu(v.z, g.slope);
                a.w = lrelu(v.w, g.slope);
            }
        }
        const f4 w = wp[(size_t)kb * 64];
        acc = mfma_k16(a, w, acc);
    }
    // D layout: lane l holds rows 4*(l/16)+q, column l%16.
    const int col = ct * kTile + (lane & 15);
    for (int q = 0; q < 4; ++q) {
        const int ro = rt * kTile + kq * 4 + q;
        if (ro < s.nrows) atomicAdd(g.out + (size_t)ro * g.ldo + col, acc[q]);
    }
}

__device__ __forceinline__ int scale_index(const float* table, int L, float s) {
    int cnt = 0;
    for (int l = 0; l < L - 1; ++l) cnt += table[l] < s ? 1 : 0;
    return cnt;
}

__global__ __launch_bounds__(256) void k_step_epilogue(StepRows s, EpiArgs e) {
    const int tid = blockIdx.x * blockDim.x + threadIdx.x;
    const int M = e.M;
    if (tid < s.nrows * M) {
        const int r = tid / M, c = tid - r * M;
        const int b = r / s.n;
        const int pos = e.order[s.ptr + (r - b * s.n)];
        const size_t lat = (size_t)b * e.H * e.W + pos;
        float* orow = e.o + (size_t)r * e.ldo;
        const float t0 = e.table[0];
        float mu;
        if (e.K == 1) {
            mu = orow[c] + e.b3[c];
            float sr = orow[M + c] + e.b3[M + c];
            orow[c] = 0.0f;
            orow[M + c] = 0.0f;
            float sg = sr > t0 ? sr : t0;
            e.scale[lat * M + c] = sg;
            e.idx[lat * M + c] = scale_index(e.table, e.L, sg);
        } else {
            float lg[3], mk[3], mx = -INFINITY;
            for (int k = 0; k < 3; ++k) {
                lg[k] = orow[k * M + c] + e.b3[k * M + c];
                mk[k] = orow[(3 + k) * M + c] + e.b3[(3 + k) * M + c];
                float sr = orow[(6 + k) * M + c] + e.b3[(6 + k) * M + c];
                orow[k * M + c] = 0.0f;
                orow[(3 + k) * M + c] = 0.0f;
                orow[(6 + k) * M + c] = 0.0f;
                float sg = sr > t0 ? sr : t0;
                const size_t q = (lat * 3 + k) * M + c;
                e.scale[q] = sg;
                e.idx[q] = scale_index(e.table, e.L, sg);
                e.cmean[q] = mk[k];
                mx = fmaxf(mx, lg[k]);
            }
            float ex[3], den = 0.0f;
            for (int k = 0; k < 3; ++k) {
                ex[k] = expf(lg[k] - mx);
                den += ex[k];
            }
            mu = 0.0f;
            for (int k = 0; k < 3; ++k) {
                float wk = ex[k] / den;
                e.weight[(lat * 3 + k) * M + c] = wk;
                mu += wk * mk[k];
            }
        }
        const size_t q = lat * M + c;
        float sv;
        if (e.encode) {
            sv = rintf(e.y[q] - mu);
            e.sym_out[q] = (int32_t)sv;
        } else {
            sv = (float)e.sym[q];
        }
        e.mean[q] = mu;
        e.y_hat[q] = sv + mu;
    }
    // Clear this step's raw sums: every product that read them has finished.
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (int u = 0; u < 3; ++u) {
        const size_t n = (size_t)s.nrows * e.clr_ld[u];
        for (size_t q = tid; q < n; q += stride) e.clr[u][q] = 0.0f;
    }
}

__global__ void k_fill_zero(float* p, size_t n) {
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t q = (size_t)blockIdx.x * blockDim.x + threadIdx.x; q < n; q += stride) p[q] = 0.0f;
}

// Grid of one product: 16x16 output tiles times k-slices, sized so that a step
// of any width offers a few thousand waves.
static dim3 gemm_grid(int nrows, int ncols, int nkb, int* kb_per_split) {
    const int tiles = ((nrows + kTile - 1) / kTile) * (ncols / kTile);
    int splits = std::max(1, std::min(nkb, 2048 / std::max(1, tiles)));
    *kb_per_split = (nkb + splits - 1) / splits;
    splits = (nkb + *kb_per_split - 1) / *kb_per_split;
    return dim3(ncols / kTile, (nrows + kTile - 1) / kTile, splits);
}

int run_steps(Plan& p, const float* psi, const int32_t* sym, const float* y, int32_t* sym_out,
              const wf_out* out, hipStream_t stream) {
    const int M = p.M;
    const size_t R = (size_t)p.max_rows;
    {
        float* bufs[4] = {p.d_ctx, p.d_h1, p.d_h2, p.d_o};
        size_t ns[4] = {R * 2 * M, R * p.Np1, R * p.Np2, R * p.n3};
        for (int u = 0; u < 4; ++u)
            hipLaunchKernelGGL(k_fill_zero, dim3(256), dim3(256), 0, stream, bufs[u], ns[u]);
    }
    GemmArgs base{};
    base.slope = p.slope;
    base.H = p.H;
    base.W = p.W;
    base.M = M;
    base.order = p.d_order;
    base.y_hat = out->y_hat;
    base.psi = psi;
    for (int k = 0; k < p.ntaps; ++k) {
        base.dy[k] = p.dy[k];
        base.dx[k] = p.dx[k];
    }
    GemmArgs gc = base, g1 = base, g2 = base, g3 = base;
    gc.wp = p.d_wc; gc.nkb = p.ntaps * M / kTile; gc.out = p.d_ctx; gc.ldo = 2 * M;
    g1.wp = p.d_w1; g1.nkb = 4 * M / kTile; g1.out = p.d_h1; g1.ldo = p.Np1;
    g1.in = p.d_ctx; g1.ldi = 2 * M; g1.in_bias = p.d_bc;
    g2.wp = p.d_w2; g2.nkb = p.Np1 / kTile; g2.out = p.d_h2; g2.ldo = p.Np2;
    g2.in = p.d_h1; g2.ldi = p.Np1; g2.in_bias = p.d_b1;
    g3.wp = p.d_w3; g3.nkb = p.Np2 / kTile; g3.out = p.d_o; g3.ldo = p.n3;
    g3.in = p.d_h2; g3.ldi = p.Np2; g3.in_bias = p.d_b2;

    EpiArgs e{};
    e.o = p.d_o; e.ldo = p.n3; e.b3 = p.d_b3; e.table = p.d_table; e.L = p.L;
    e.M = M; e.K = p.K; e.H = p.H; e.W = p.W; e.order = p.d_order;
    e.sym = sym; e.y = y; e.sym_out = sym_out; e.encode = y != nullptr;
    e.y_hat = out->y_hat; e.mean = out->mean; e.scale = out->scale; e.idx = out->idx;
    e.weight = out->weight; e.cmean = out->comp_mean;
    e.clr[0] = p.d_ctx; e.clr_ld[0] = 2 * M;
    e.clr[1] = p.d_h1; e.clr_ld[1] = p.Np1;
    e.clr[2] = p.d_h2; e.clr_ld[2] = p.Np2;

    for (int t = 0; t < p.T; ++t) {
        StepRows s{p.step_n[t], p.step_ptr[t], p.B * p.step_n[t]};
        dim3 grid = gemm_grid(s.nrows, 2 * M, gc.nkb, &gc.kb_per_split);
        hipLaunchKernelGGL(k_step_gemm<A_TAPS>, grid, dim3(64), 0, stream, s, gc);
        grid = gemm_grid(s.nrows, p.Np1, g1.nkb, &g1.kb_per_split);
        hipLaunchKernelGGL(k_step_gemm<A_PSI_CTX>, grid, dim3(64), 0, stream, s, g1);
        grid = gemm_grid(s.nrows, p.Np2, g2.nkb, &g2.kb_per_split);
        hipLaunchKernelGGL(k_step_gemm<A_HIDDEN>, grid, dim3(64), 0, stream, s, g2);
        grid = gemm_grid(s.nrows, p.n3, g3.nkb, &g3.kb_per_split);
        hipLaunchKernelGGL(k_step_gemm<A_HIDDEN>, grid, dim3(64), 0, stream, s, g3);
        const int n = s.nrows * M;
        hipLaunchKernelGGL(k_step_epilogue, dim3((n + 255) / 256), dim3(256), 0, stream, s, e);
    }
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(WF_E_HIP, std::string("kernel launch: ") + hipGetErrorString(err));
    return WF_OK;
}

}  // namespace wf
