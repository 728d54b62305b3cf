// The transforms around the autoregressive decode (the latent pipeline of
// Sec. II-A): the hyper-decoder h_s (z_hat -> the hyperprior half psi of the
// entropy parameters) and the synthesis transform g_s (y_hat -> image), for
// an end-to-end decode timing with random weights.  Layer list (the paper
// names the models, not their layers; this is the mean-scale hyperprior model
// of the family the workloads are named after):
//   h_s: transposed conv 5x5 s2 (N -> M), ReLU; transposed conv 5x5 s2
//        (M -> 3M/2), ReLU; conv 3x3 s1 (3M/2 -> 2M), cropped to the H x W grid
//   g_s: 3 x (transposed conv 5x5 s2, inverse GDN) (M -> N -> N -> N), then
//        transposed conv 5x5 s2 (N -> 3)
//
// Every layer is one implicit-GEMM kernel on MFMA.  A stride-2 transposed
// conv (padding 2, output padding 1) splits into four output parity classes
// (oy mod 2, ox mod 2); class (py, px) is an ordinary product over the taps
// ky = py + 2 ty, kx = px + 2 tx, reading input pixel (qy + 1 - ty, qx + 1 - tx)
// for output pixel (2 qy + py, 2 qx + px).  Rows of the product are the class's
// output pixels, columns the output channels, k the (tap, input channel)
// pairs, tap-major.  Inverse GDN is the same product over the channels of
// the squared input, x_c sqrt(beta_c + sum_j gamma_cj x_j^2), with gamma^T
// as the weight panel.  Weights are packed per layer and class in the operand
// order of the step kernels.  A transposed conv with at most 4 output
// channels (the image's 3) puts all four classes into the columns instead:
// rows are input pixels, columns (class, channel), k the 3x3 input
// neighbourhood (taps a class does not use have zero weights), so one
// 16-column tile carries all 12 outputs of an input pixel.
#include <cmath>
#include <vector>

#include "wf_device.h"
#include "wf_pack.h"

namespace wf {

enum { XM_DECONV = 0, XM_CONV3 = 1, XM_GDN = 2, XM_DECONV4 = 3 };

struct ConvArgs {
    const float* in;
    float* out;
    const void* wp[4];        // packed panel per output class
    const float* bias;        // [Co] (deconv, conv)
    const float* beta;        // [Co] (GDN)
    int B, Hi, Wi, Ci;        // input [B][Hi][Wi][Ci]
    int Hq, Wq;               // output pixels of one class per image (rows = B Hq Wq)
    int Co, Cop;              // output channels, and padded to whole column tiles
    int Ho, Wo;               // output array [B][Ho][Wo][Co]; pixels outside are not stored
    int relu;
};

// Rows: RTW row tiles per wave, 4 / WCOL waves along the rows; columns: CTW
// column tiles per wave, WCOL waves along the columns.
template <int RTW, int CTW, int WCOL>
struct ConvShape {
    static constexpr int kRowTiles = RTW * (4 / WCOL), kColTiles = CTW * WCOL;
};

template <class P, int MODE, int RTW, int CTW, int WCOL>
__global__ __launch_bounds__(kThreads) void k_conv(ConvArgs a) {
    using A = typename P::A;
    using Bw = typename P::B;
    using S = ConvShape<RTW, CTW, WCOL>;
    constexpr int KB = RTW == 4 || P::kBf16 ? 6 : 8;   // k-blocks in flight per wave
    const int cls = blockIdx.z, py = cls >> 1, px = cls & 1;
    const int nky = MODE == XM_DECONV ? (py ? 2 : 3) : (MODE == XM_GDN ? 1 : 3);
    const int nkx = MODE == XM_DECONV ? (px ? 2 : 3) : (MODE == XM_GDN ? 1 : 3);
    const int cbn = a.Ci / P::kK;                        // k-blocks per tap
    const int nkb = nky * nkx * cbn;
    const int nrows = a.B * a.Hq * a.Wq, nct = a.Cop / kTile;
    const int ncb = (nct + S::kColTiles - 1) / S::kColTiles;
    const int cb = blockIdx.x % ncb, rb = blockIdx.x / ncb;
    const int wave = wave_id(), lane = threadIdx.x & 63, kq = lane >> 4;
    const int wr = wave / WCOL, wc = wave % WCOL;
    const int rt0 = rb * S::kRowTiles + wr * RTW, ct0 = cb * S::kColTiles + wc * CTW;
    if (rt0 * kTile >= nrows) return;                    // (whole wave past the rows; no barrier below)

    int rb_[RTW], ry[RTW], rx[RTW];
    bool rv[RTW];
#pragma unroll
    for (int i = 0; i < RTW; ++i) {
        const int r = (rt0 + i) * kTile + (lane & 15);
        rv[i] = r < nrows;
        const int rr = rv[i] ? r : 0;
        rb_[i] = rr / (a.Hq * a.Wq);
        const int rem = rr - rb_[i] * a.Hq * a.Wq;
        ry[i] = rem / a.Wq;
        rx[i] = rem - ry[i] * a.Wq;
    }
    const Bw* w[CTW];
    bool cv[CTW];
#pragma unroll
    for (int j = 0; j < CTW; ++j) {
        cv[j] = ct0 + j < nct;                           // wave-uniform
        w[j] = static_cast<const Bw*>(a.wp[cls]) + (size_t)(cv[j] ? ct0 + j : 0) * nkb * 64 + lane;
    }
    auto la = [&](int i, int kb) -> A {
        const int t = kb / cbn;
        const int c0 = (kb - t * cbn) * P::kK + kq * (P::kK / 4);
        int dy = 0, dx = 0;
        if (MODE == XM_DECONV) {
            const int ty = t / nkx;
            dy = 1 - ty;
            dx = 1 - (t - ty * nkx);
        } else if (MODE == XM_CONV3 || MODE == XM_DECONV4) {
            const int ty = t / 3;
            dy = ty - 1;
            dx = t - ty * 3 - 1;
        }
        const int iy = ry[i] + dy, ix = rx[i] + dx;
        const bool ok = rv[i] && iy >= 0 && iy < a.Hi && ix >= 0 && ix < a.Wi;
        const size_t q = (((size_t)rb_[i] * a.Hi + iy) * a.Wi + ix) * a.Ci + c0;
        if constexpr (P::kBf16) {
            f4 u = ld4<false>(a.in, q, ok), v = ld4<false>(a.in, q + 4, ok);
            if (MODE == XM_GDN) {
                u = u * u;
                v = v * v;
            }
            return split8(u, v);
        } else {
            f4 u = ld4<false>(a.in, q, ok);
            if (MODE == XM_GDN) u = u * u;
            return u;
        }
    };
    f4 acc[RTW][CTW];
#pragma unroll
    for (int i = 0; i < RTW; ++i)
#pragma unroll
        for (int j = 0; j < CTW; ++j) acc[i][j] = zero4();
    for (int kc = 0; kc < nkb; kc += KB) {
        A av[KB][RTW];
        Bw bv[KB][CTW];
#pragma unroll
        for (int u = 0; u < KB; ++u) {
            const int k = min(kc + u, nkb - 1);
#pragma unroll
            for (int i = 0; i < RTW; ++i) av[u][i] = la(i, k);
#pragma unroll
            for (int j = 0; j < CTW; ++j) bv[u][j] = w[j][(size_t)k * 64];
        }
#pragma unroll
        for (int u = 0; u < KB; ++u)
            if (kc + u < nkb)
#pragma unroll
                for (int i = 0; i < RTW; ++i)
#pragma unroll
                    for (int j = 0; j < CTW; ++j) acc[i][j] = P::mma(av[u][i], bv[u][j], acc[i][j]);
    }
    // lane holds rows 4*(lane/16) + q of each row tile, column lane%16
#pragma unroll
    for (int j = 0; j < CTW; ++j) {
        const int cc = (ct0 + j) * kTile + (lane & 15);   // column: channel, or (class, channel)
        const int ccls = MODE == XM_DECONV4 ? cc / a.Co : 0;
        const int c = MODE == XM_DECONV4 ? cc - ccls * a.Co : cc;
        if (!cv[j] || c >= a.Co || ccls >= 4) continue;
        const float add = MODE == XM_GDN ? a.beta[c] : a.bias[c];
#pragma unroll
        for (int i = 0; i < RTW; ++i)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int ro = (rt0 + i) * kTile + kq * 4 + q;
                if (ro >= nrows) continue;
                const int b = ro / (a.Hq * a.Wq), rem = ro - b * a.Hq * a.Wq;
                const int qy = rem / a.Wq, qx = rem - qy * a.Wq;
                int oy = qy, ox = qx;
                if (MODE == XM_DECONV) {
                    oy = 2 * qy + py;
                    ox = 2 * qx + px;
                } else if (MODE == XM_DECONV4) {
                    oy = 2 * qy + (ccls >> 1);
                    ox = 2 * qx + (ccls & 1);
                }
                if (oy >= a.Ho || ox >= a.Wo) continue;
                float v = acc[i][j][q] + add;
                if (MODE == XM_GDN) {
                    v = a.in[(((size_t)b * a.Hi + qy) * a.Wi + qx) * a.Ci + c] * sqrtf(v);
                } else if (a.relu) {
                    v = fmaxf(v, 0.0f);
                }
                a.out[(((size_t)b * a.Ho + oy) * a.Wo + ox) * a.Co + c] = v;
            }
    }
}

// ---- plan -------------------------------------------------------------------

struct Layer {
    int mode, Ci, Co, Cop, relu;
    const void* wp[4];
    const float* bias;
    const float* beta;
};

struct Xform {
    int N, M, B, H, W, Hz, Wz, precision;
    int device = 0;
    std::vector<void*> owned;
    Layer hs[3], gs[4], gdn[3];
    float *hs_a = nullptr, *hs_b = nullptr, *g_a = nullptr, *g_b = nullptr;
};

static int xf_fail_hip(hipError_t e, const char* what) {
    return fail(WF_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

template <class T>
static int xf_upload(Xform* x, const T** dst, const std::vector<T>& v) {
    T* p = nullptr;
    hipError_t e = hipMalloc((void**)&p, v.size() * sizeof(T));
    if (e != hipSuccess) return fail(WF_E_NOMEM, std::string("transform weights: ") + hipGetErrorString(e));
    x->owned.push_back(p);
    e = hipMemcpy(p, v.data(), v.size() * sizeof(T), hipMemcpyHostToDevice);
    if (e != hipSuccess) return xf_fail_hip(e, "transform weights");
    *dst = p;
    return WF_OK;
}

static int xf_alloc(Xform* x, float** dst, size_t n) {
    hipError_t e = hipMalloc((void**)dst, n * sizeof(float));
    if (e != hipSuccess) return fail(WF_E_NOMEM, std::string("transform workspace: ") + hipGetErrorString(e));
    x->owned.push_back(*dst);
    return WF_OK;
}

// Pack one layer: wt(k, n) of class c over k = (tap, input channel), tap-major.
template <class F>
static int xf_pack(Xform* x, Layer& L, int nclass, F wt) {
    const bool bf = x->precision == WF_BF16;
    for (int c = 0; c < nclass; ++c) {
        const int py = c >> 1, px = c & 1;
        const int nky = L.mode == XM_DECONV ? (py ? 2 : 3) : (L.mode == XM_GDN ? 1 : 3);
        const int nkx = L.mode == XM_DECONV ? (px ? 2 : 3) : (L.mode == XM_GDN ? 1 : 3);
        const int K = nky * nkx * L.Ci;
        auto f = [&](int k, int n) { return wt(c, k / L.Ci, nkx, k % L.Ci, n); };
        const int ncol = L.mode == XM_DECONV4 ? 4 * L.Co : L.Co;   // columns that carry weights
        int rc = bf ? xf_upload(x, reinterpret_cast<const uint16_t**>(&L.wp[c]), pack_panel_bf16(K, ncol, K, L.Cop, f))
                    : xf_upload(x, reinterpret_cast<const float**>(&L.wp[c]), pack_panel(K, ncol, K, L.Cop, f));
        if (rc != WF_OK) return rc;
    }
    for (int c = nclass; c < 4; ++c) L.wp[c] = L.wp[0];
    return WF_OK;
}

// Transposed conv weight W[ci][co][5][5]: tap t of class (py, px) is
// (ky, kx) = (py + 2 (t / nkx), px + 2 (t % nkx)).
static int xf_deconv(Xform* x, Layer& L, const float* w, const float* b, int Ci, int Co, int relu) {
    L.mode = XM_DECONV; L.Ci = Ci; L.Co = Co; L.Cop = (Co + kTile - 1) / kTile * kTile; L.relu = relu;
    int rc = xf_pack(x, L, 4, [&](int c, int t, int nkx, int ci, int co) {
        const int ky = (c >> 1) + 2 * (t / nkx), kx = (c & 1) + 2 * (t % nkx);
        return w[(((size_t)ci * Co + co) * 5 + ky) * 5 + kx];
    });
    if (rc != WF_OK) return rc;
    return xf_upload(x, &L.bias, std::vector<float>(b, b + Co));
}

// All four classes in the columns (Co <= 4): column n = class * Co + co, tap
// (dy, dx) = (t / 3 - 1, t % 3 - 1) of the input neighbourhood, which class
// (py, px) reaches through (ky, kx) = (py + 2 - 2 dy, px + 2 - 2 dx) when both
// are at most 4 (zero weight otherwise).
static int xf_deconv4(Xform* x, Layer& L, const float* w, const float* b, int Ci, int Co) {
    L.mode = XM_DECONV4; L.Ci = Ci; L.Co = Co; L.Cop = (4 * Co + kTile - 1) / kTile * kTile; L.relu = 0;
    int rc = xf_pack(x, L, 1, [&](int, int t, int, int ci, int n) -> float {
        const int cls = n / Co, co = n - cls * Co;
        const int ky = (cls >> 1) + 2 - 2 * (t / 3 - 1), kx = (cls & 1) + 2 - 2 * (t % 3 - 1);
        if (ky > 4 || kx > 4) return 0.0f;
        return w[(((size_t)ci * Co + co) * 5 + ky) * 5 + kx];
    });
    if (rc != WF_OK) return rc;
    return xf_upload(x, &L.bias, std::vector<float>(b, b + Co));
}

static int xf_conv3(Xform* x, Layer& L, const float* w, const float* b, int Ci, int Co) {
    L.mode = XM_CONV3; L.Ci = Ci; L.Co = Co; L.Cop = (Co + kTile - 1) / kTile * kTile; L.relu = 0;
    int rc = xf_pack(x, L, 1, [&](int, int t, int, int ci, int co) {
        return w[(((size_t)co * Ci + ci) * 3 + t / 3) * 3 + t % 3];
    });
    if (rc != WF_OK) return rc;
    return xf_upload(x, &L.bias, std::vector<float>(b, b + Co));
}

static int xf_gdn(Xform* x, Layer& L, const float* beta, const float* gamma, int C) {
    L.mode = XM_GDN; L.Ci = C; L.Co = C; L.Cop = (C + kTile - 1) / kTile * kTile; L.relu = 0;
    int rc = xf_pack(x, L, 1, [&](int, int, int, int j, int c) { return gamma[(size_t)c * C + j]; });
    if (rc != WF_OK) return rc;
    return xf_upload(x, &L.beta, std::vector<float>(beta, beta + C));
}

template <class P, int MODE>
static void launch_layer(const Layer& L, const float* in, float* out, int B, int Hi, int Wi, int Hq, int Wq, int Ho,
                         int Wo, hipStream_t st) {
    ConvArgs a{};
    a.in = in; a.out = out; a.bias = L.bias; a.beta = L.beta;
    for (int c = 0; c < 4; ++c) a.wp[c] = L.wp[c];
    a.B = B; a.Hi = Hi; a.Wi = Wi; a.Ci = L.Ci; a.Hq = Hq; a.Wq = Wq;
    a.Co = L.Co; a.Cop = L.Cop; a.Ho = Ho; a.Wo = Wo; a.relu = L.relu;
    const int nrows = B * Hq * Wq, nct = L.Cop / kTile, ncls = MODE == XM_DECONV ? 4 : 1;
    // Row tiles per wave: 4 with fp32 operands (each weight operand then feeds
    // four MFMA chains, which halves the weight reads against 2); bf16 pairs
    // already hold twice the registers per operand and keep 2 (measured:
    // 4 was 5% slower there).
    constexpr int RTW = P::kBf16 ? 2 : 4;
    if (nct <= 1) {   // narrow output (the image's 3 channels): 4 RTW row tiles x 1 column tile per workgroup
        using S = ConvShape<RTW, 1, 1>;
        const int nb = ((nrows + S::kRowTiles * kTile - 1) / (S::kRowTiles * kTile)) * nct;
        hipLaunchKernelGGL((k_conv<P, MODE, RTW, 1, 1>), dim3(nb, 1, ncls), dim3(kThreads), 0, st, a);
    } else {          // 2 RTW row tiles x 4 column tiles per workgroup
        using S = ConvShape<RTW, 2, 2>;
        const int nb = ((nrows + S::kRowTiles * kTile - 1) / (S::kRowTiles * kTile)) *
                       ((nct + S::kColTiles - 1) / S::kColTiles);
        hipLaunchKernelGGL((k_conv<P, MODE, RTW, 2, 2>), dim3(nb, 1, ncls), dim3(kThreads), 0, st, a);
    }
}

template <class P>
static void run_layer(const Layer& L, const float* in, float* out, int B, int Hi, int Wi, int Ho, int Wo,
                      hipStream_t st) {
    if (L.mode == XM_DECONV) launch_layer<P, XM_DECONV>(L, in, out, B, Hi, Wi, Hi, Wi, Ho, Wo, st);
    else if (L.mode == XM_CONV3) launch_layer<P, XM_CONV3>(L, in, out, B, Hi, Wi, Ho, Wo, Ho, Wo, st);
    else if (L.mode == XM_DECONV4) launch_layer<P, XM_DECONV4>(L, in, out, B, Hi, Wi, Hi, Wi, Ho, Wo, st);
    else launch_layer<P, XM_GDN>(L, in, out, B, Hi, Wi, Hi, Wi, Hi, Wi, st);
}

template <class P>
static void hyper(const Xform& x, const float* z, float* psi, hipStream_t st) {
    const int B = x.B, Hz = x.Hz, Wz = x.Wz;
    run_layer<P>(x.hs[0], z, x.hs_a, B, Hz, Wz, 2 * Hz, 2 * Wz, st);
    run_layer<P>(x.hs[1], x.hs_a, x.hs_b, B, 2 * Hz, 2 * Wz, 4 * Hz, 4 * Wz, st);
    run_layer<P>(x.hs[2], x.hs_b, psi, B, 4 * Hz, 4 * Wz, x.H, x.W, st);   // cropped to the latent grid
}

template <class P>
static void synth(const Xform& x, const float* y, float* img, hipStream_t st) {
    const int B = x.B;
    int h = x.H, w = x.W;
    const float* in = y;
    for (int k = 0; k < 3; ++k) {
        run_layer<P>(x.gs[k], in, x.g_a, B, h, w, 2 * h, 2 * w, st);
        h *= 2;
        w *= 2;
        run_layer<P>(x.gdn[k], x.g_a, x.g_b, B, h, w, h, w, st);
        in = x.g_b;
    }
    run_layer<P>(x.gs[3], in, img, B, h, w, 2 * h, 2 * w, st);
}

static void free_xform(Xform* x) {
    if (!x) return;
    for (void* p : x->owned)
        if (p) (void)hipFree(p);
    delete x;
}

}  // namespace wf

using namespace wf;

extern "C" {

int wf_xform_plan(const wf_xform_desc* d, wf_xform_t* out) {
    if (!out) return fail(WF_E_INVALID, "out is NULL");
    *out = nullptr;
    if (!d) return fail(WF_E_INVALID, "desc is NULL");
    if (d->N < 1 || d->M < 1 || d->B < 1 || d->H < 1 || d->W < 1)
        return fail(WF_E_INVALID, "N, M, B, H and W must be positive");
    if (d->precision != WF_FP32 && d->precision != WF_BF16) return fail(WF_E_INVALID, "unknown precision");
    if (!d->hs_w[0] || !d->hs_w[1] || !d->hs_w[2] || !d->hs_b[0] || !d->hs_b[1] || !d->hs_b[2])
        return fail(WF_E_INVALID, "a hyper-decoder weight pointer is NULL");
    for (int k = 0; k < 4; ++k)
        if (!d->gs_w[k] || !d->gs_b[k] || (k < 3 && (!d->gdn_beta[k] || !d->gdn_gamma[k])))
            return fail(WF_E_INVALID, "a synthesis weight pointer is NULL");
    const int kb = d->precision == WF_BF16 ? 32 : kTile;
    if (d->N % kb || d->M % kb || (d->M * 3 / 2) % kb || d->M % 2)
        return fail(WF_E_UNSUPPORTED, "N, M and 3M/2 must be multiples of the k-block (16 fp32, 32 bf16)");
    const long long big = (long long)d->B * 8 * d->H * 8 * d->W * d->N * 4;
    const long long lat = (long long)d->B * d->H * d->W * (long long)(d->M > 2 * d->M ? d->M : 2 * d->M) * 4;
    if (big >= kBufBytes || lat >= kBufBytes || (long long)d->B * 4 * ((d->H + 3) / 4) * 4 * ((d->W + 3) / 4) *
                                                     (d->M * 3 / 2) * 4 >= kBufBytes)
        return fail(WF_E_UNSUPPORTED, "transform activations exceed the 2 GiB buffer window");
    Xform* x = new (std::nothrow) Xform();
    if (!x) return fail(WF_E_NOMEM, "host allocation");
    x->N = d->N; x->M = d->M; x->B = d->B; x->H = d->H; x->W = d->W;
    x->Hz = (d->H + 3) / 4; x->Wz = (d->W + 3) / 4; x->precision = d->precision;
    hipError_t e = hipGetDevice(&x->device);
    int rc = e == hipSuccess ? WF_OK : xf_fail_hip(e, "hipGetDevice");
    const int N = d->N, M = d->M, C = M * 3 / 2;
    if (rc == WF_OK) rc = xf_deconv(x, x->hs[0], d->hs_w[0], d->hs_b[0], N, M, 1);
    if (rc == WF_OK) rc = xf_deconv(x, x->hs[1], d->hs_w[1], d->hs_b[1], M, C, 1);
    if (rc == WF_OK) rc = xf_conv3(x, x->hs[2], d->hs_w[2], d->hs_b[2], C, 2 * M);
    const int gi[4] = {M, N, N, N}, go[4] = {N, N, N, 3};
    for (int k = 0; k < 4 && rc == WF_OK; ++k) {
        rc = go[k] <= 4 ? xf_deconv4(x, x->gs[k], d->gs_w[k], d->gs_b[k], gi[k], go[k])
                        : xf_deconv(x, x->gs[k], d->gs_w[k], d->gs_b[k], gi[k], go[k], 0);
        if (rc == WF_OK && k < 3) rc = xf_gdn(x, x->gdn[k], d->gdn_beta[k], d->gdn_gamma[k], N);
    }
    const size_t B = d->B;
    if (rc == WF_OK) rc = xf_alloc(x, &x->hs_a, B * 2 * x->Hz * 2 * x->Wz * M);
    if (rc == WF_OK) rc = xf_alloc(x, &x->hs_b, B * 4 * x->Hz * 4 * x->Wz * C);
    if (rc == WF_OK) rc = xf_alloc(x, &x->g_a, B * 8 * d->H * 8 * d->W * N);
    if (rc == WF_OK) rc = xf_alloc(x, &x->g_b, B * 8 * d->H * 8 * d->W * N);
    if (rc != WF_OK) {
        free_xform(x);
        return rc;
    }
    *out = reinterpret_cast<wf_xform_t>(x);
    return WF_OK;
}

int wf_hyper_synthesis(wf_xform_t plan, const float* z_hat, float* psi, hipStream_t stream) {
    if (!plan || !z_hat || !psi) return fail(WF_E_INVALID, "plan, z_hat or psi is NULL");
    const Xform& x = *reinterpret_cast<Xform*>(plan);
    if (x.precision == WF_BF16) hyper<PBF16>(x, z_hat, psi, stream);
    else hyper<PF32>(x, z_hat, psi, stream);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? WF_OK : xf_fail_hip(e, "transform launch");
}

int wf_synthesis(wf_xform_t plan, const float* y_hat, float* image, hipStream_t stream) {
    if (!plan || !y_hat || !image) return fail(WF_E_INVALID, "plan, y_hat or image is NULL");
    const Xform& x = *reinterpret_cast<Xform*>(plan);
    if (x.precision == WF_BF16) synth<PBF16>(x, y_hat, image, stream);
    else synth<PF32>(x, y_hat, image, stream);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? WF_OK : xf_fail_hip(e, "transform launch");
}

void wf_xform_destroy(wf_xform_t plan) { free_xform(reinterpret_cast<Xform*>(plan)); }

}  // extern "C"
