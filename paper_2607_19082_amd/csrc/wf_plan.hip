// Host side of libwf: argument validation, the wavefront schedule, weight
// repacking into MFMA tile order, plan lifetime and the C entry points.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <type_traits>

#include "wf_internal.h"
#include "wf_pack.h"

namespace wf {

static thread_local std::string g_err;

int fail(int code, const std::string& msg) {
    g_err = msg;
    return code;
}

#define WF_HIP(call)                                                              \
    do {                                                                          \
        hipError_t e_ = (call);                                                   \
        if (e_ != hipSuccess)                                                     \
            return fail(WF_E_HIP, std::string(#call) + ": " + hipGetErrorString(e_)); \
    } while (0)

// Radius R of a mask's (2R+1)x(2R+1) kernel, or -1 for an unknown mask.
static int mask_radius(int mask) {
    switch (mask) {
    case WF_MASK_3X3: return 1;
    case WF_MASK_FULL:
    case WF_MASK_RELAXED: return 2;
    case WF_MASK_7X7: return 3;
    default: return -1;
    }
}

// Causal taps of a mask in kernel raster order (Appendix A, Def. 1): the R
// rows above with |dx| <= R, then the R latents to the left.  The relaxed 5x5
// mask drops (-2,+2) and (-1,+2).
static int mask_taps(int mask, int* dy, int* dx) {
    const int R = mask_radius(mask);
    int n = 0;
    for (int y = -R; y <= 0; ++y) {
        for (int x = -R; x <= R; ++x) {
            if (y == 0 && x >= 0) continue;
            if (mask == WF_MASK_RELAXED && x == 2 && (y == -1 || y == -2)) continue;
            dy[n] = y;
            dx[n] = x;
            ++n;
        }
    }
    return n;
}

// Shear of the schedule of a W-wide grid: the mask's least shear, or W when
// the grid is narrower.  Then every latent depends on its raster predecessor
// (through (0,-1), or (-1, W-1) for the first of a row: W - 1 < lambda - 1 = R),
// so the raster order t = W*i + j is the earliest-possible schedule.
static int schedule_shear(int lam, int W) { return W < lam ? W : lam; }

// Least integer shear lambda >= 0 with lambda*di + dj > 0 for every
// dependence vector d = (-dy, -dx) of the taps (Sec. III-B, Eq. 6-7).
static int least_shear(int ntaps, const int* dy, const int* dx) {
    for (int lam = 0; lam < 64; ++lam) {
        bool ok = true;
        for (int k = 0; k < ntaps; ++k)
            if (lam * (-dy[k]) + (-dx[k]) <= 0) ok = false;
        if (ok) return lam;
    }
    return -1;
}

static int round_up(int v, int m) { return (v + m - 1) / m * m; }
static int round16(int v) { return round_up(v, kTile); }
// k-block of the packed operands: 16 values of k for fp32, 32 for bf16
static int kblock(int precision) { return precision == WF_BF16 ? 32 : 16; }
// columns of one job's column group (kC tiles of 16): d1, d2 are padded to it
static int colgroup(int precision) { return kTile * (precision == WF_BF16 ? kColsBf16 : kColsF32); }
static int padded(int d, int precision) { return round_up(round_up(d, kblock(precision)), colgroup(precision)); }

static int check_desc(const wf_desc* d) {
    if (!d) return fail(WF_E_INVALID, "desc is NULL");
    if (d->H < 1 || d->W < 1 || d->M < 1 || d->B < 1)
        return fail(WF_E_INVALID, "H, W, M and B must be positive");
    if (d->K != 1 && d->K != 3) return fail(WF_E_INVALID, "K must be 1 or 3");
    if (d->d1 < 1 || d->d2 < 1) return fail(WF_E_INVALID, "d1 and d2 must be positive");
    if (mask_radius(d->mask) < 0) return fail(WF_E_INVALID, "unknown mask");
    if (d->precision != WF_FP32 && d->precision != WF_BF16)
        return fail(WF_E_INVALID, "unknown precision");
    if (d->driver < WF_DRIVER_STREAM || d->driver > WF_DRIVER_RESIDENT)
        return fail(WF_E_INVALID, "unknown driver");
    if (!d->ctx_w || !d->ctx_b || !d->w1 || !d->b1 || !d->w2 || !d->b2 || !d->w3 || !d->b3 ||
        !d->scale_table)
        return fail(WF_E_INVALID, "a weight or table pointer is NULL");
    if (d->L < 2 || d->L > kMaxTable) return fail(WF_E_INVALID, "L must be in [2, 256]");
    for (int l = 0; l < d->L; ++l) {
        float t = d->scale_table[l];
        if (!(t > 0.0f) || !std::isfinite(t)) return fail(WF_E_INVALID, "scale table must be positive");
        if (l > 0 && !(t > d->scale_table[l - 1]))
            return fail(WF_E_INVALID, "scale table must be strictly increasing");
    }
    if (!std::isfinite(d->lrelu_slope)) return fail(WF_E_INVALID, "lrelu_slope must be finite");
    if (d->group < 0) return fail(WF_E_INVALID, "group must be >= 0");
    if (d->param_order != WF_ORDER_NATIVE && d->param_order != WF_ORDER_SCALES_FIRST)
        return fail(WF_E_INVALID, "unknown param_order");
    if (d->entropy_coder != WF_EC_NONE && d->entropy_coder != WF_EC_RANS)
        return fail(WF_E_INVALID, "unknown entropy_coder");
    if (d->entropy_coder == WF_EC_RANS) {
        if (d->group > 1) return fail(WF_E_UNSUPPORTED, "entropy coding needs the exact decode (group <= 1)");
        if (d->driver != WF_DRIVER_STREAM && d->driver != WF_DRIVER_GRAPH)
            return fail(WF_E_UNSUPPORTED, "entropy coding needs the stream or graph driver");
    }
    if (d->group > 1 && d->driver != WF_DRIVER_STREAM && d->driver != WF_DRIVER_GRAPH)
        return fail(WF_E_UNSUPPORTED, "context approximation (group > 1) needs the stream or graph driver");
    if (d->M % kTile != 0) return fail(WF_E_UNSUPPORTED, "M must be a multiple of 16");
    if (d->cu_limit < 0) return fail(WF_E_INVALID, "cu_limit must be >= 0");
    int dy[kMaxTaps], dx[kMaxTaps];
    int nt = mask_taps(d->mask, dy, dx);
    int lam = least_shear(nt, dy, dx);
    if (d->W < lam && d->group > 1)
        return fail(WF_E_UNSUPPORTED, "context approximation needs W at least the shear factor (Thm. 1)");
    // every array the kernels read through raw buffer instructions (psi, y_hat,
    // the per-step activations) must fit the buffer window
    const long long lat = (long long)d->B * d->H * d->W;
    if (lat * 2 * d->M * 4 >= kBufBytes || lat * padded(d->d1, d->precision) * 4 >= kBufBytes ||
        lat * 3 * d->M > (1LL << 31) - 1)
        return fail(WF_E_UNSUPPORTED, "problem too large for the 2 GiB buffer window");
    // a k-block of the tap gathers must not straddle two taps
    if (d->M % kblock(d->precision) != 0) return fail(WF_E_UNSUPPORTED, "bf16 operands need M a multiple of 32");
    return WF_OK;
}

template <class T>
static int upload(Plan* p, T** dst, const T* src, size_t n) {
    WF_HIP(hipMalloc((void**)dst, n * sizeof(T)));
    p->owned.push_back((void*)*dst);
    WF_HIP(hipMemcpy(*dst, src, n * sizeof(T), hipMemcpyHostToDevice));
    return WF_OK;
}

template <class T>
static int alloc(Plan* p, T** dst, size_t n) {
    WF_HIP(hipMalloc((void**)dst, n * sizeof(T)));
    p->owned.push_back((void*)*dst);
    return WF_OK;
}

static void free_plan(Plan* p) {
    if (!p) return;
    if (p->graph_exec) (void)hipGraphExecDestroy(p->graph_exec);
    if (p->graph) (void)hipGraphDestroy(p->graph);
    if (p->graph_exec_ec) (void)hipGraphExecDestroy(p->graph_exec_ec);
    if (p->graph_ec) (void)hipGraphDestroy(p->graph_ec);
    if (p->cap_stream) (void)hipStreamDestroy(p->cap_stream);
    for (void* q : p->owned)
        if (q) (void)hipFree(q);
    delete p;
}

// Folded layer-1 weights of one tap: F[c][n] = sum_o W1[n][2M + o] * Wc[o][c][tap]
// (fp64 accumulation), for c < M, n < d1; with `bf` both factors are the
// bf16-rounded weights.
static void fold_tap(const wf_desc* d, int dy, int dx, bool bf, std::vector<double>& out) {
    const int M = d->M, d1 = d->d1, R = mask_radius(d->mask), kw = 2 * R + 1;
    auto q = [bf](float v) { return (double)(bf ? bf16_value_of(v) : v); };
    std::vector<double> wc((size_t)2 * M * M);
    for (int o = 0; o < 2 * M; ++o)
        for (int c = 0; c < M; ++c)
            wc[(size_t)o * M + c] = q(d->ctx_w[(((size_t)o * M + c) * kw + (dy + R)) * kw + (dx + R)]);
    out.assign((size_t)M * d1, 0.0);
    std::vector<double> acc(M);
    for (int n = 0; n < d1; ++n) {
        std::fill(acc.begin(), acc.end(), 0.0);
        const float* w1b = d->w1 + (size_t)n * 4 * M + 2 * M;
        for (int o = 0; o < 2 * M; ++o) {
            const double w = q(w1b[o]);
            const double* row = &wc[(size_t)o * M];
            for (int c = 0; c < M; ++c) acc[c] += w * row[c];
        }
        for (int c = 0; c < M; ++c) out[(size_t)c * d1 + n] = acc[c];
    }
}

// geometry_only: stop after the schedule, the tap split and the step
// arguments (host only; nothing is allocated on the device).
static int build_plan(const wf_desc* d, Plan* p, bool geometry_only = false) {
    p->H = d->H; p->W = d->W; p->M = d->M; p->B = d->B; p->K = d->K;
    p->d1 = d->d1; p->d2 = d->d2; p->n3 = (d->K == 1 ? 2 : 9) * d->M;
    p->mask = d->mask; p->precision = d->precision; p->driver = d->driver;
    p->L = d->L; p->slope = d->lrelu_slope;
    p->cu_limit = d->cu_limit;
    p->ntaps = mask_taps(d->mask, p->dy, p->dx);
    p->lambda = schedule_shear(least_shear(p->ntaps, p->dy, p->dx), d->W);
    const int H = p->H, W = p->W, M = p->M, lam = p->lambda;
    p->T = W + lam * (H - 1);
    p->group = d->group > 1 ? d->group : 1;
    p->steps = (p->T + p->group - 1) / p->group;

    // Wavefront steps: the latents with lambda*i + j == t; a step's rows are
    // its latents by ascending grid row, image-major.
    p->step_of.resize((size_t)H * W);
    std::vector<int> step_n(p->T, 0);
    for (int i = 0; i < H; ++i)
        for (int j = 0; j < W; ++j) {
            const int t = lam * i + j;
            p->step_of[(size_t)i * W + j] = t;
            step_n[t]++;
        }
    int maxn = 0;
    for (int t = 0; t < p->T; ++t) maxn = std::max(maxn, step_n[t]);
    p->max_rows = round16(p->B * maxn);   // whole 16-row tiles (tiled activation arrays)
    // Grouped decode: group g holds the latents with floor(t / N) == g, listed
    // by image, grid row and column.
    std::vector<int32_t> rowlat;
    if (p->group > 1) {
        const int N = p->group;
        p->g_r0.assign(p->steps, 0);
        p->g_n.assign(p->steps, 0);
        rowlat.reserve((size_t)p->B * H * W);
        int maxg = 0;
        for (int g = 0; g < p->steps; ++g) {
            p->g_r0[g] = (int)rowlat.size();
            for (int b = 0; b < p->B; ++b)
                for (int i = 0; i < H; ++i)
                    for (int j = std::max(0, g * N - lam * i); j < W && lam * i + j < (g + 1) * N; ++j)
                        rowlat.push_back((int32_t)(((size_t)b * H + i) * W + j));
            p->g_n[g] = (int)rowlat.size() - p->g_r0[g];
            maxg = std::max(maxg, p->g_n[g]);
        }
        if (rowlat.size() != (size_t)p->B * H * W) return fail(WF_E_UNSUPPORTED, "internal: group rows do not cover the grid");
        p->max_rows = round16(maxg);
    }
    for (size_t q = 0; q < p->step_of.size() && p->group > 1; ++q) p->step_of[q] /= p->group;
    const bool bf = p->precision == WF_BF16;
    p->Np1 = padded(p->d1, p->precision);
    p->Np2 = padded(p->d2, p->precision);
    p->nph = 3;
    const int d1 = p->d1, Np1 = p->Np1;

    StepArgs& a = p->args;
    a = StepArgs{};
    a.H = H; a.W = W; a.M = M; a.B = p->B; a.K = p->K; a.L = p->L; a.lambda = lam;
    a.Np1 = Np1; a.Np2 = p->Np2; a.n3 = p->n3; a.slope = p->slope; a.max_rows = p->max_rows;
    a.group = p->group;
    const int R = mask_radius(d->mask), kw = 2 * R + 1;
    a.R = R;
    a.row_w = d->mask == WF_MASK_RELAXED ? 4 : kw;
    a.gparts = (M / kblock(p->precision) + kJobWaves - 1) / kJobWaves;   // one channel chunk per wave of a part

    // Split the taps by age (delta = steps between producer and consumer).
    // On a grid narrower than the mask's shear, taps of the rows above at
    // dx >= W never lie in the grid; the exact decode leaves them out.
    std::vector<int> new_taps, old_taps;
    for (int k = 0; k < p->ntaps; ++k) {
        if (p->dy[k] < 0 && p->dx[k] >= W) continue;
        const int delta = lam * (-p->dy[k]) - p->dx[k];
        if (delta < 1) return fail(WF_E_UNSUPPORTED, "internal: a tap is not decoded before its consumer");
        (delta == 1 ? new_taps : old_taps).push_back(k);
    }
    if ((int)new_taps.size() != kMaxNew) return fail(WF_E_UNSUPPORTED, "mask must have two taps of age one");
    a.ctx_parts = p->driver == WF_DRIVER_DATAFLOW ? kDfCtxParts : (bf ? kCtxPartsBf16 : kCtxPartsF32);
    a.n_old = (int)old_taps.size();
    if (R > kMaxRadius) return fail(WF_E_UNSUPPORTED, "internal: mask radius too large");
    int cnt[kMaxRadius + 1] = {};
    for (int o : old_taps) cnt[p->dy[o] + R]++;
    for (int q = 0, first = 0; q < kMaxRadius; ++q) {
        first += cnt[q];
        a.old_start[q] = q < R ? first : 1 << 30;
    }
    a.new_dx0 = p->dx[new_taps[0]];
    // the kernels rebuild every tap from these scalars: check that they can
    for (int o = 0; o < a.n_old; ++o) {
        int row = 0;
        while (row < kMaxRadius && o >= a.old_start[row]) ++row;
        const int first = row == 0 ? 0 : a.old_start[row - 1];
        if (p->dy[old_taps[o]] != row - R || p->dx[old_taps[o]] != o - first - R)
            return fail(WF_E_UNSUPPORTED, "old taps are not row-contiguous from dx = -R");
    }
    for (int k = 0; k < p->ntaps; ++k) {
        const int up = R * a.row_w;
        const int dy = k < up ? k / a.row_w - R : 0;
        const int dx = k < up ? k % a.row_w - R : k - up - R;
        if (p->dy[k] != dy || p->dx[k] != dx) return fail(WF_E_UNSUPPORTED, "internal: mask is not raster-contiguous");
    }
    if (p->dy[new_taps[0]] != -1 || p->dy[new_taps[1]] != 0 || p->dx[new_taps[1]] != -1)
        return fail(WF_E_UNSUPPORTED, "unexpected new taps");
    if (geometry_only) return WF_OK;

    WF_HIP(hipGetDevice(&p->device));
    int rc;

    float* f;
    // upload a packed panel after checking that it holds exactly the
    // (column tile, k-block) lane operands the kernels read from it
    const int kbk = kblock(p->precision);
    auto put = [&](const void** dst, int cols, int kdim, const auto& v) -> int {
        using T = typename std::decay_t<decltype(v)>::value_type;
        if (kdim % kbk != 0 || v.size() != (size_t)(cols / kTile) * (kdim / kbk) * 64 * (16 / sizeof(T)))
            return fail(WF_E_UNSUPPORTED, "internal: packed panel does not match the kernels' tiling");
        T* q = nullptr;
        int r = upload(p, &q, v.data(), v.size());
        *dst = q;
        return r;
    };
    auto wc_of = [&](const std::vector<int>& taps) {
        return [&, taps](int k, int n) {
            const int o = k / M, c = k % M;
            return d->ctx_w[(((size_t)n * M + c) * kw + (p->dy[taps[o]] + R)) * kw + (p->dx[taps[o]] + R)];
        };
    };
    // all taps, channel-chunk-major k (chunk of kb channels, then the taps):
    // the grouped decode's context product
    auto wc_all = [&](int k, int n) {
        const int per = kbk * p->ntaps;
        const int q = k / per, rem = k - q * per, tap = rem / kbk, c = q * kbk + rem % kbk;
        return d->ctx_w[(((size_t)n * M + c) * kw + (p->dy[tap] + R)) * kw + (p->dx[tap] + R)];
    };
    if (p->group > 1) {
        const int ka = p->ntaps * M;
        rc = bf ? put(&a.wp_all, 2 * M, ka, pack_panel_bf16(ka, 2 * M, ka, 2 * M, wc_all))
                : put(&a.wp_all, 2 * M, ka, pack_panel(ka, 2 * M, ka, 2 * M, wc_all));
        if (rc != WF_OK) return rc;
        int32_t* rl = nullptr;
        if ((rc = upload(p, &rl, rowlat.data(), rowlat.size())) != WF_OK) return rc;
        a.rowlat = rl;
    }
    auto w1a = [&](int k, int n) { return d->w1[(size_t)n * 4 * M + k]; };
    auto w1b = [&](int k, int n) { return d->w1[(size_t)n * 4 * M + 2 * M + k]; };
    auto w2f = [&](int k, int n) { return d->w2[(size_t)n * d1 + k]; };
    // the last layer's rows in the native block order
    std::vector<int> row3(p->n3);
    {
        const int nb = p->K == 1 ? 2 : 3, bs = p->n3 / nb;   // blocks of bs rows
        for (int b = 0; b < nb; ++b)
            for (int r = 0; r < bs; ++r)
                row3[b * bs + r] = (d->param_order == WF_ORDER_SCALES_FIRST ? nb - 1 - b : b) * bs + r;
    }
    std::vector<float> b3(p->n3);
    for (int n = 0; n < p->n3; ++n) b3[n] = d->b3[row3[n]];
    auto w3f = [&](int k, int n) { return d->w3[(size_t)row3[n] * p->d2 + k]; };
    // Fold the new taps' conv into the context half of layer 1, and the
    // context bias into the hoisted part (bf16: from the bf16 weights).
    std::vector<float> b_hoist(Np1, 0.0f);
    std::vector<std::vector<double>> fold(kMaxNew);
    for (int k = 0; k < kMaxNew; ++k) fold_tap(d, p->dy[new_taps[k]], p->dx[new_taps[k]], bf, fold[k]);
    for (int n = 0; n < d1; ++n) {
        double acc = d->b1[n];
        const float* w1r = d->w1 + (size_t)n * 4 * M + 2 * M;
        for (int o = 0; o < 2 * M; ++o) acc += (double)(bf ? bf16_value_of(w1r[o]) : w1r[o]) * (double)d->ctx_b[o];
        b_hoist[n] = (float)acc;
    }
    if (bf) {
        const int kn = kMaxNew * M, ko = a.n_old * M, Np2 = p->Np2, n3 = p->n3;
        // the folded block as a pair: hi = bf16(F), lo = bf16(F - hi)
        auto f_hi = [&](int k, int n) { return (float)fold[k / M][(size_t)(k % M) * d1 + n]; };
        auto f_lo = [&](int k, int n) {
            const double v = fold[k / M][(size_t)(k % M) * d1 + n];
            return (float)(v - (double)bf16_value_of((float)v));
        };
        if ((rc = put(&a.wp_hoist, Np1, 2 * M, pack_panel_bf16(2 * M, d1, 2 * M, Np1, w1a))) != WF_OK) return rc;
        if ((rc = put(&a.wp_l1, Np1, 2 * M, pack_panel_bf16(2 * M, d1, 2 * M, Np1, w1b))) != WF_OK) return rc;
        if ((rc = put(&a.wp_new, Np1, kn, pack_panel_bf16(kn, d1, kn, Np1, f_hi))) != WF_OK) return rc;
        if ((rc = put(&a.wp_new_lo, Np1, kn, pack_panel_bf16(kn, d1, kn, Np1, f_lo))) != WF_OK) return rc;
        fold.clear();
        if ((rc = put(&a.wp_old, 2 * M, ko, pack_panel_bf16(ko, 2 * M, ko, 2 * M, wc_of(old_taps)))) != WF_OK) return rc;
        if ((rc = put(&a.wp2, Np2, Np1, pack_panel_bf16(d1, p->d2, Np1, Np2, w2f))) != WF_OK) return rc;
        if ((rc = put(&a.wp3, n3, Np2, pack_panel_bf16(p->d2, n3, Np2, n3, w3f))) != WF_OK) return rc;
    } else {
        const int knew = kMaxNew * M;
        const int ko = a.n_old * M, Np2 = p->Np2, n3 = p->n3;
        if ((rc = put(&a.wp_hoist, Np1, 2 * M, pack_panel(2 * M, d1, 2 * M, Np1, w1a))) != WF_OK) return rc;
        if ((rc = put(&a.wp_l1, Np1, knew + 2 * M, pack_panel(knew + 2 * M, d1, knew + 2 * M, Np1, [&](int k, int n) {
                 if (k < knew) return (float)fold[k / M][(size_t)(k % M) * d1 + n];
                 return w1b(k - knew, n);
             }))) != WF_OK)
            return rc;
        fold.clear();
        if ((rc = put(&a.wp_old, 2 * M, ko, pack_panel(ko, 2 * M, ko, 2 * M, wc_of(old_taps)))) != WF_OK) return rc;
        if ((rc = put(&a.wp2, Np2, Np1, pack_panel(d1, p->d2, Np1, Np2, w2f))) != WF_OK) return rc;
        if ((rc = put(&a.wp3, n3, Np2, pack_panel(p->d2, n3, Np2, n3, w3f))) != WF_OK) return rc;
    }
    std::vector<float> b2(p->Np2, 0.0f);
    std::copy(d->b2, d->b2 + p->d2, b2.begin());
    if ((rc = upload(p, &f, b_hoist.data(), b_hoist.size())) != WF_OK) return rc;
    a.b_hoist = f;
    if ((rc = upload(p, &f, b2.data(), b2.size())) != WF_OK) return rc;
    a.b2 = f;
    if ((rc = upload(p, &f, b3.data(), b3.size())) != WF_OK) return rc;
    a.b3 = f;
    if ((rc = upload(p, &f, d->scale_table, (size_t)p->L)) != WF_OK) return rc;
    a.table = f;

    const size_t MR = (size_t)p->max_rows;
    const size_t nlat = (size_t)p->B * H * W;
    float *h1 = nullptr, *h2 = nullptr;
    if ((rc = alloc(p, &h1, MR * Np1)) != WF_OK) return rc;
    if ((rc = alloc(p, &h2, MR * p->Np2)) != WF_OK) return rc;
    a.h1 = h1;
    a.h2 = h2;
    a.h2b = h2;
    if (p->driver == WF_DRIVER_DATAFLOW) {
        // the dataflow driver double-buffers layer 2's output by step parity
        float* h2b = nullptr;
        if ((rc = alloc(p, &h2b, MR * p->Np2)) != WF_OK) return rc;
        a.h2b = h2b;
    }
    if ((rc = alloc(p, &a.p1, nlat * Np1)) != WF_OK) return rc;
    const int nparts = std::max(kCtxPartsMax, p->group > 1 ? a.gparts : 0);
    if ((rc = alloc(p, &a.ctxo, (size_t)2 * nparts * MR * 2 * M)) != WF_OK) return rc;
    if (bf) {
        if ((rc = alloc(p, &a.ybf, nlat * 2 * M)) != WF_OK) return rc;
    }
    if ((rc = alloc(p, &p->d_call, 1)) != WF_OK) return rc;
    WF_HIP(hipMemset(p->d_call, 0, sizeof(CallPtrs)));
    a.cp = p->d_call;
    if ((rc = alloc(p, &p->d_err, 1)) != WF_OK) return rc;
    WF_HIP(hipMemset(p->d_err, 0, sizeof(int)));
    // one round of jobs: the persistent grid (two workgroups per CU); the
    // per-step kernels have the same residency
    if ((rc = persistent_grid(*p, &a.slots)) != WF_OK) return rc;
    if (p->driver == WF_DRIVER_PERSISTENT) {
        p->grid = a.slots;
        if ((rc = alloc(p, &p->d_bar, kBarrierWords)) != WF_OK) return rc;
        WF_HIP(hipMemset(p->d_bar, 0, kBarrierWords * sizeof(unsigned)));
    }
    if (p->driver == WF_DRIVER_DATAFLOW) {
        std::vector<int2> lists;
        if ((rc = build_dataflow(*p, lists, p->df)) != WF_OK) return rc;
        int2* jobs = nullptr;
        if ((rc = upload(p, &jobs, lists.data(), lists.size())) != WF_OK) return rc;
        p->df.jobs = jobs;
        if ((rc = alloc(p, &p->df.cnt, p->df.cnt_words)) != WF_OK) return rc;
        if ((rc = coop_grid(*p, dataflow_fn(*p), &p->grid)) != WF_OK) return rc;
        // half of the grid runs the critical chain (one workgroup per CU when
        // two fit), the other half the old-tap context
        p->df.ncrit = p->grid >= 2 * kXcds ? p->grid / 2 / kXcds * kXcds : p->grid;
        if (p->df.ncrit == p->grid) return fail(WF_E_UNSUPPORTED, "dataflow driver needs at least 16 workgroups");
    }
    if (p->driver == WF_DRIVER_RESIDENT && (rc = build_resident(*p)) != WF_OK) return rc;
    if (d->entropy_coder == WF_EC_RANS && (rc = build_ec(p, d->scale_table, d->L)) != WF_OK) return rc;
    WF_HIP(hipDeviceSynchronize());

    if (p->driver == WF_DRIVER_GRAPH) {
        // Capture every kernel of one call once; calls only republish their
        // pointers to d_call and replay the graph.
        WF_HIP(hipStreamCreateWithFlags(&p->cap_stream, hipStreamNonBlocking));
        WF_HIP(hipStreamBeginCapture(p->cap_stream, hipStreamCaptureModeThreadLocal));
        int erc = enqueue_steps(*p, p->cap_stream);
        hipGraph_t g = nullptr;
        hipError_t e = hipStreamEndCapture(p->cap_stream, &g);
        if (erc != WF_OK) {
            if (g) (void)hipGraphDestroy(g);
            return erc;
        }
        if (e != hipSuccess) return fail(WF_E_HIP, std::string("graph capture: ") + hipGetErrorString(e));
        p->graph = g;
        WF_HIP(hipGraphInstantiate(&p->graph_exec, p->graph, nullptr, nullptr, 0));
        if (p->ec) {
            // the decode from streams: the same steps with the entropy-decoding phase C
            WF_HIP(hipStreamBeginCapture(p->cap_stream, hipStreamCaptureModeThreadLocal));
            erc = enqueue_steps(*p, p->cap_stream, true);
            g = nullptr;
            e = hipStreamEndCapture(p->cap_stream, &g);
            if (erc != WF_OK) {
                if (g) (void)hipGraphDestroy(g);
                return erc;
            }
            if (e != hipSuccess) return fail(WF_E_HIP, std::string("graph capture: ") + hipGetErrorString(e));
            p->graph_ec = g;
            WF_HIP(hipGraphInstantiate(&p->graph_exec_ec, p->graph_ec, nullptr, nullptr, 0));
        }
    }
    return WF_OK;
}

}  // namespace wf

using namespace wf;

extern "C" {

const char* wf_last_error(void) { return g_err.c_str(); }

int wf_schedule(int32_t H, int32_t W, int32_t mask, int32_t* step_of, int32_t* n_steps,
                int32_t* lambda_out) {
    if (H < 1 || W < 1) return fail(WF_E_INVALID, "H and W must be positive");
    if (mask_radius(mask) < 0) return fail(WF_E_INVALID, "unknown mask");
    if (!n_steps) return fail(WF_E_INVALID, "n_steps is NULL");
    int dy[kMaxTaps], dx[kMaxTaps];
    int nt = mask_taps(mask, dy, dx);
    const int lam = schedule_shear(least_shear(nt, dy, dx), W);
    if (step_of)
        for (int i = 0; i < H; ++i)
            for (int j = 0; j < W; ++j) step_of[(size_t)i * W + j] = lam * i + j;
    *n_steps = W + lam * (H - 1);
    if (lambda_out) *lambda_out = lam;
    return WF_OK;
}

int wf_validate(const wf_desc* desc) { return check_desc(desc); }

int wf_plan(const wf_desc* desc, wf_plan_t* out) {
    if (!out) return fail(WF_E_INVALID, "out is NULL");
    *out = nullptr;
    int rc = check_desc(desc);
    if (rc != WF_OK) return rc;
    Plan* p = new (std::nothrow) Plan();
    if (!p) return fail(WF_E_NOMEM, "host allocation failed");
    try {
        rc = build_plan(desc, p);
    } catch (const std::bad_alloc&) {
        rc = fail(WF_E_NOMEM, "host allocation failed");
    }
    if (rc != WF_OK) {
        free_plan(p);
        return rc;
    }
    *out = reinterpret_cast<wf_plan_t>(p);
    return WF_OK;
}

int wf_plan_deps(const wf_desc* desc, int32_t* out, int64_t capacity, int64_t* needed) {
    if (!needed) return fail(WF_E_INVALID, "needed is NULL");
    int rc = check_desc(desc);
    if (rc != WF_OK) return rc;
    if (desc->driver != WF_DRIVER_DATAFLOW && desc->driver != WF_DRIVER_RESIDENT)
        return fail(WF_E_UNSUPPORTED, "dependency lists exist for the dataflow and resident drivers");
    if (capacity < 0) return fail(WF_E_INVALID, "negative capacity");
    Plan p;
    std::vector<int32_t> v;
    try {
        rc = build_plan(desc, &p, true);
        if (rc == WF_OK) rc = desc->driver == WF_DRIVER_DATAFLOW ? dataflow_deps(p, v) : resident_deps(p, v);
    } catch (const std::bad_alloc&) {
        rc = fail(WF_E_NOMEM, "host allocation failed");
    }
    if (rc != WF_OK) return rc;
    *needed = (int64_t)v.size();
    if (out) {
        if (capacity < (int64_t)v.size()) return fail(WF_E_INVALID, "out holds fewer entries than needed");
        std::copy(v.begin(), v.end(), out);
    }
    return WF_OK;
}

int wf_plan_set_waits(wf_plan_t plan, int64_t spin_budget_ticks, int32_t stall) {
    if (!plan) return fail(WF_E_INVALID, "plan is NULL");
    if (stall != 0 && stall != 1) return fail(WF_E_INVALID, "stall must be 0 or 1");
    Plan* p = reinterpret_cast<Plan*>(plan);
    p->spin_budget = spin_budget_ticks > 0 ? spin_budget_ticks : 100000000;
    p->stall = stall;
    return WF_OK;
}

int wf_plan_schedule(wf_plan_t plan, int32_t* step_of, int32_t* n_steps) {
    if (!plan || !n_steps) return fail(WF_E_INVALID, "plan or n_steps is NULL");
    Plan* p = reinterpret_cast<Plan*>(plan);
    if (step_of) std::copy(p->step_of.begin(), p->step_of.end(), step_of);
    *n_steps = p->steps;
    return WF_OK;
}

static int check_out(const Plan* p, const wf_out* out) {
    if (!out || !out->y_hat || !out->mean || !out->scale || !out->idx)
        return fail(WF_E_INVALID, "y_hat, mean, scale and idx outputs are required");
    if (p->K == 3 && (!out->weight || !out->comp_mean))
        return fail(WF_E_INVALID, "weight and comp_mean outputs are required for K = 3");
    // the resident driver reads y_hat with ordinary cached loads while it is
    // being written: its rows must be whole 128-byte lines (M is a multiple
    // of 32 there, so the base must be aligned)
    if (p->driver == WF_DRIVER_RESIDENT && reinterpret_cast<uintptr_t>(out->y_hat) % 128 != 0)
        return fail(WF_E_INVALID, "the resident driver needs y_hat aligned to 128 bytes");
    return WF_OK;
}

static int run_call(Plan* p, const CallPtrs& c, hipStream_t stream, bool ec = false) {
    int rc = enqueue_set_call(*p, c, stream);
    if (rc != WF_OK) return rc;
    if (p->driver == WF_DRIVER_GRAPH) {
        WF_HIP(hipGraphLaunch(ec ? p->graph_exec_ec : p->graph_exec, stream));
        return WF_OK;
    }
    if (ec) return enqueue_steps(*p, stream, true);
    if (p->driver == WF_DRIVER_PERSISTENT) return enqueue_persistent(*p, stream);
    if (p->driver == WF_DRIVER_DATAFLOW) return enqueue_dataflow(*p, stream);
    if (p->driver == WF_DRIVER_RESIDENT) return enqueue_resident(*p, stream);
    return enqueue_steps(*p, stream);
}

static CallPtrs call_ptrs(const float* psi, const int32_t* sym, const float* y, int32_t* sym_out,
                          const wf_out* out) {
    CallPtrs c{};
    c.psi = psi; c.sym = sym; c.y = y; c.sym_out = sym_out; c.encode = y != nullptr;
    c.y_hat = out->y_hat; c.mean = out->mean; c.scale = out->scale; c.idx = out->idx;
    c.weight = out->weight; c.cmean = out->comp_mean;
    return c;
}

// the plan's entropy-decoding state in a call's pointers
static void ec_ptrs(const Plan* p, CallPtrs& c, const uint32_t* bits) {
    c.bits = bits;
    c.ec_x = p->ec_x; c.ec_pos = p->ec_pos; c.ec_end = p->ec_end;
    c.ec_n = p->ec_n; c.ec_base = p->ec_base; c.ec_cum = p->ec_cum; c.ec_lut = p->ec_lut;
    c.mix_X = p->mix_X; c.mix_base = p->mix_base; c.mix_G = p->mix_G;
    c.err = p->d_err;
}

int wf_decode(wf_plan_t plan, const float* psi, const int32_t* sym, const wf_out* out,
              hipStream_t stream) {
    if (!plan || !psi || !sym) return fail(WF_E_INVALID, "plan, psi or sym is NULL");
    Plan* p = reinterpret_cast<Plan*>(plan);
    int rc = check_out(p, out);
    if (rc != WF_OK) return rc;
    return run_call(p, call_ptrs(psi, sym, nullptr, nullptr, out), stream);
}

int wf_encode(wf_plan_t plan, const float* psi, const float* y, int32_t* sym_out,
              const wf_out* out, hipStream_t stream) {
    if (!plan || !psi || !y || !sym_out) return fail(WF_E_INVALID, "plan, psi, y or sym_out is NULL");
    Plan* p = reinterpret_cast<Plan*>(plan);
    int rc = check_out(p, out);
    if (rc != WF_OK) return rc;
    return run_call(p, call_ptrs(psi, nullptr, y, sym_out, out), stream);
}

int wf_encode_bits(wf_plan_t plan, const float* psi, const float* y, int32_t* sym_out, const wf_out* out,
                   uint32_t* bits, int64_t bits_capacity, uint32_t* offsets, hipStream_t stream) {
    if (!plan || !psi || !y || !sym_out || !bits || !offsets)
        return fail(WF_E_INVALID, "plan, psi, y, sym_out, bits or offsets is NULL");
    Plan* p = reinterpret_cast<Plan*>(plan);
    if (!p->ec) return fail(WF_E_UNSUPPORTED, "the plan was built without entropy coding");
    if (bits_capacity < 0) return fail(WF_E_INVALID, "negative capacity");
    int rc = check_out(p, out);
    if (rc != WF_OK) return rc;
    if ((rc = run_call(p, call_ptrs(psi, nullptr, y, sym_out, out), stream)) != WF_OK) return rc;
    return enqueue_ec_encode(*p, sym_out, *out, bits, bits_capacity, offsets, stream);
}

int wf_decode_bits(wf_plan_t plan, const float* psi, const uint32_t* bits, int64_t n_words, const uint32_t* offsets,
                   int32_t* sym_out, const wf_out* out, hipStream_t stream) {
    if (!plan || !psi || !bits || !offsets || !sym_out)
        return fail(WF_E_INVALID, "plan, psi, bits, offsets or sym_out is NULL");
    Plan* p = reinterpret_cast<Plan*>(plan);
    if (!p->ec) return fail(WF_E_UNSUPPORTED, "the plan was built without entropy coding");
    if (n_words < 0) return fail(WF_E_INVALID, "negative word count");
    int rc = check_out(p, out);
    if (rc != WF_OK) return rc;
    if ((rc = enqueue_ec_init(*p, bits, n_words, offsets, stream)) != WF_OK) return rc;
    CallPtrs c = call_ptrs(psi, nullptr, nullptr, sym_out, out);
    ec_ptrs(p, c, bits);
    return run_call(p, c, stream, true);
}

int wf_plan_trace(wf_plan_t plan, int64_t* stamps, int64_t capacity, int64_t* needed, int32_t* grid) {
    if (!plan) return fail(WF_E_INVALID, "plan is NULL");
    Plan* p = reinterpret_cast<Plan*>(plan);
    if (p->driver != WF_DRIVER_PERSISTENT && p->driver != WF_DRIVER_DATAFLOW && p->driver != WF_DRIVER_RESIDENT)
        return fail(WF_E_UNSUPPORTED, "tracing needs the persistent, dataflow or resident driver");
    if (stamps && capacity < 0) return fail(WF_E_INVALID, "negative capacity");
    p->stamps = reinterpret_cast<long long*>(stamps);
    p->stamps_cap = stamps ? capacity : 0;
    if (p->driver == WF_DRIVER_RESIDENT) {
        // three entries per task of every workgroup
        if (needed) *needed = 3LL * p->res.ntasks * p->grid;
        if (grid) *grid = p->grid;
        return WF_OK;
    }
    if (p->driver == WF_DRIVER_DATAFLOW) {
        // three entries per job of the plan's job lists
        if (needed) *needed = 3LL * p->df.off[2 * kXcds];
        if (grid) *grid = p->grid;
        return WF_OK;
    }
    // barriers: the prologue (two with fp32) and one per phase of every step
    const int64_t pro = 2;
    if (needed) *needed = (int64_t)(pro + p->nph * (int64_t)p->T) * (p->grid + 1);
    if (grid) *grid = p->grid;
    return WF_OK;
}

int wf_measure_floor(wf_plan_t plan, float* node_us, float* barrier_us) {
    if (!plan || !node_us || !barrier_us) return fail(WF_E_INVALID, "plan or an output is NULL");
    return measure_floor(*reinterpret_cast<Plan*>(plan), node_us, barrier_us);
}

int wf_plan_sync(wf_plan_t plan, hipStream_t stream) {
    if (!plan) return fail(WF_E_INVALID, "plan is NULL");
    Plan* p = reinterpret_cast<Plan*>(plan);
    WF_HIP(hipStreamSynchronize(stream));
    int err = 0;
    WF_HIP(hipMemcpy(&err, p->d_err, sizeof(int), hipMemcpyDeviceToHost));
    if (err) {
        WF_HIP(hipMemset(p->d_err, 0, sizeof(int)));
        if (err == kErrStream) return fail(WF_E_STREAM, "a malformed rANS stream (or a scale level out of range)");
        if (err == kErrCapacity) return fail(WF_E_CAPACITY, "the encoded streams exceed the bits buffer");
        return fail(WF_E_TIMEOUT, "a device-wide wait exceeded its spin budget");
    }
    return WF_OK;
}

void wf_plan_destroy(wf_plan_t plan) { free_plan(reinterpret_cast<Plan*>(plan)); }

}  // extern "C"
