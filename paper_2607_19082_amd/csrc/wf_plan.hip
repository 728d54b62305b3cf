// Host side of libwf: argument validation, the wavefront schedule, weight
// repacking into MFMA tile order, plan lifetime and the C entry points.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>

#include "wf_internal.h"

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

// Causal taps of the 5x5 mask in kernel raster order (Appendix A, Def. 1,
// R = 2): the two rows above with |dx| <= 2, then the two latents to the left.
// The relaxed mask drops (-2,+2) and (-1,+2).
static int mask_taps(int mask, int* dy, int* dx) {
    int n = 0;
    for (int y = -2; y <= 0; ++y) {
        for (int x = -2; x <= 2; ++x) {
            if (y == 0 && x >= 0) continue;
            if (mask == WF_MASK_RELAXED && x == 2 && (y == -1 || y == -2)) continue;
            dy[n] = y;
            dx[n] = x;
            ++n;
        }
    }
    return n;
}

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

static int check_desc(const wf_desc* d) {
    if (!d) return fail(WF_E_INVALID, "desc is NULL");
    if (d->H < 1 || d->W < 1 || d->M < 1 || d->B < 1)
        return fail(WF_E_INVALID, "H, W, M and B must be positive");
    if (d->K != 1 && d->K != 3) return fail(WF_E_INVALID, "K must be 1 or 3");
    if (d->d1 < 1 || d->d2 < 1) return fail(WF_E_INVALID, "d1 and d2 must be positive");
    if (d->mask != WF_MASK_FULL && d->mask != WF_MASK_RELAXED)
        return fail(WF_E_INVALID, "unknown mask");
    if (d->precision != WF_FP32 && d->precision != WF_BF16)
        return fail(WF_E_INVALID, "unknown precision");
    if (d->driver < WF_DRIVER_STREAM || d->driver > WF_DRIVER_PERSISTENT)
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
    if (d->M % kTile != 0) return fail(WF_E_UNSUPPORTED, "M must be a multiple of 16");
    int dy[kMaxTaps], dx[kMaxTaps];
    int nt = mask_taps(d->mask, dy, dx);
    int lam = least_shear(nt, dy, dx);
    if (d->W < lam) return fail(WF_E_UNSUPPORTED, "W must be at least the shear factor (Thm. 1)");
    const long long lat = (long long)d->B * d->H * d->W;
    if (lat * 2 * d->M > (1LL << 31) - 1 || lat * 3 * d->M > (1LL << 31) - 1)
        return fail(WF_E_UNSUPPORTED, "problem too large for 32-bit element indexing");
    if (d->precision == WF_BF16) return fail(WF_E_UNSUPPORTED, "bf16 operands are not built yet");
    if (d->driver != WF_DRIVER_STREAM) return fail(WF_E_UNSUPPORTED, "driver not built yet");
    return WF_OK;
}

static int round16(int v) { return (v + kTile - 1) / kTile * kTile; }

// Pack Wt[k][n] (k < K, n < N; zero beyond) into the MFMA operand order used
// by the step kernels: for column tile ct and k-block kb (16 values of k),
// lane l holds Wt[kb*16 + (l/16)*4 + q][ct*16 + l%16] for q = 0..3.
template <class F>
static std::vector<float> pack_panel(int K, int N, F wt) {
    const int Kp = round16(K), Np = round16(N);
    const int nkb = Kp / kTile;
    std::vector<float> out((size_t)Np * Kp, 0.0f);
    for (int ct = 0; ct < Np / kTile; ++ct)
        for (int kb = 0; kb < nkb; ++kb)
            for (int l = 0; l < 64; ++l)
                for (int q = 0; q < 4; ++q) {
                    int k = kb * kTile + (l / 16) * 4 + q;
                    int n = ct * kTile + l % 16;
                    float v = (k < K && n < N) ? wt(k, n) : 0.0f;
                    out[(((size_t)ct * nkb + kb) * 64 + l) * 4 + q] = v;
                }
    return out;
}

template <class T>
static int upload(T** dst, const T* src, size_t n) {
    WF_HIP(hipMalloc((void**)dst, n * sizeof(T)));
    WF_HIP(hipMemcpy(*dst, src, n * sizeof(T), hipMemcpyHostToDevice));
    return WF_OK;
}

static void free_plan(Plan* p) {
    if (!p) return;
    void* ptrs[] = {p->d_order, p->d_wc, p->d_w1, p->d_w2, p->d_w3, p->d_bc, p->d_b1,
                    p->d_b2, p->d_b3, p->d_table, p->d_ctx, p->d_h1, p->d_h2, p->d_o, p->d_err};
    for (void* q : ptrs)
        if (q) (void)hipFree(q);
    delete p;
}

static int build_plan(const wf_desc* d, Plan* p) {
    p->H = d->H; p->W = d->W; p->M = d->M; p->B = d->B; p->K = d->K;
    p->d1 = d->d1; p->d2 = d->d2; p->n3 = (d->K == 1 ? 2 : 9) * d->M;
    p->mask = d->mask; p->precision = d->precision; p->driver = d->driver;
    p->L = d->L; p->slope = d->lrelu_slope;
    p->ntaps = mask_taps(d->mask, p->dy, p->dx);
    p->lambda = least_shear(p->ntaps, p->dy, p->dx);
    const int H = p->H, W = p->W, M = p->M;
    p->T = W + p->lambda * (H - 1);

    // Wavefront step lists: positions with lambda*i + j == t, by ascending row.
    p->step_of.resize((size_t)H * W);
    p->step_ptr.assign(p->T, 0);
    p->step_n.assign(p->T, 0);
    for (int i = 0; i < H; ++i)
        for (int j = 0; j < W; ++j) {
            int t = p->lambda * i + j;
            p->step_of[(size_t)i * W + j] = t;
            p->step_n[t]++;
        }
    std::vector<int> order((size_t)H * W);
    int maxn = 0;
    for (int t = 0, acc = 0; t < p->T; ++t) {
        p->step_ptr[t] = acc;
        acc += p->step_n[t];
        maxn = std::max(maxn, p->step_n[t]);
    }
    {
        std::vector<int> fill(p->T, 0);
        for (int i = 0; i < H; ++i)
            for (int j = 0; j < W; ++j) {
                int t = p->lambda * i + j;
                order[p->step_ptr[t] + fill[t]++] = i * W + j;
            }
    }
    p->max_rows = p->B * maxn;
    p->Np1 = round16(p->d1);
    p->Np2 = round16(p->d2);

    WF_HIP(hipGetDevice(&p->device));
    int rc;
    if ((rc = upload(&p->d_order, order.data(), order.size())) != WF_OK) return rc;

    // Context conv as a GEMM over the causal taps: k = tap*M + c, n = output channel.
    const int Kc = p->ntaps * M;
    auto wc = pack_panel(Kc, 2 * M, [&](int k, int n) {
        int tap = k / M, c = k % M;
        return d->ctx_w[(((size_t)n * M + c) * 5 + (p->dy[tap] + 2)) * 5 + (p->dx[tap] + 2)];
    });
    auto w1 = pack_panel(4 * M, p->d1, [&](int k, int n) { return d->w1[(size_t)n * 4 * M + k]; });
    auto w2 = pack_panel(p->d1, p->d2, [&](int k, int n) { return d->w2[(size_t)n * p->d1 + k]; });
    auto w3 = pack_panel(p->d2, p->n3, [&](int k, int n) { return d->w3[(size_t)n * p->d2 + k]; });
    if ((rc = upload(&p->d_wc, wc.data(), wc.size())) != WF_OK) return rc;
    if ((rc = upload(&p->d_w1, w1.data(), w1.size())) != WF_OK) return rc;
    if ((rc = upload(&p->d_w2, w2.data(), w2.size())) != WF_OK) return rc;
    if ((rc = upload(&p->d_w3, w3.data(), w3.size())) != WF_OK) return rc;

    std::vector<float> b1(p->Np1, 0.0f), b2(p->Np2, 0.0f);
    std::copy(d->b1, d->b1 + p->d1, b1.begin());
    std::copy(d->b2, d->b2 + p->d2, b2.begin());
    if ((rc = upload(&p->d_bc, d->ctx_b, (size_t)2 * M)) != WF_OK) return rc;
    if ((rc = upload(&p->d_b1, b1.data(), b1.size())) != WF_OK) return rc;
    if ((rc = upload(&p->d_b2, b2.data(), b2.size())) != WF_OK) return rc;
    if ((rc = upload(&p->d_b3, d->b3, (size_t)p->n3)) != WF_OK) return rc;
    if ((rc = upload(&p->d_table, d->scale_table, (size_t)p->L)) != WF_OK) return rc;

    const size_t R = (size_t)p->max_rows;
    WF_HIP(hipMalloc((void**)&p->d_ctx, R * 2 * M * sizeof(float)));
    WF_HIP(hipMalloc((void**)&p->d_h1, R * p->Np1 * sizeof(float)));
    WF_HIP(hipMalloc((void**)&p->d_h2, R * p->Np2 * sizeof(float)));
    WF_HIP(hipMalloc((void**)&p->d_o, R * p->n3 * sizeof(float)));
    WF_HIP(hipMalloc((void**)&p->d_err, sizeof(int)));
    WF_HIP(hipMemset(p->d_err, 0, sizeof(int)));
    WF_HIP(hipDeviceSynchronize());
    return WF_OK;
}

}  // namespace wf

using namespace wf;

extern "C" {

const char* wf_last_error(void) { return g_err.c_str(); }

int wf_schedule(int32_t H, int32_t W, int32_t mask, int32_t* step_of, int32_t* n_steps,
                int32_t* lambda_out) {
    if (H < 1 || W < 1) return fail(WF_E_INVALID, "H and W must be positive");
    if (mask != WF_MASK_FULL && mask != WF_MASK_RELAXED) return fail(WF_E_INVALID, "unknown mask");
    if (!n_steps) return fail(WF_E_INVALID, "n_steps is NULL");
    int dy[kMaxTaps], dx[kMaxTaps];
    int nt = mask_taps(mask, dy, dx);
    int lam = least_shear(nt, dy, dx);
    if (W < lam) return fail(WF_E_UNSUPPORTED, "W must be at least the shear factor (Thm. 1)");
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

int wf_plan_schedule(wf_plan_t plan, int32_t* step_of, int32_t* n_steps) {
    if (!plan || !n_steps) return fail(WF_E_INVALID, "plan or n_steps is NULL");
    Plan* p = reinterpret_cast<Plan*>(plan);
    if (step_of) std::copy(p->step_of.begin(), p->step_of.end(), step_of);
    *n_steps = p->T;
    return WF_OK;
}

static int check_out(const Plan* p, const wf_out* out) {
    if (!out || !out->y_hat || !out->mean || !out->scale || !out->idx)
        return fail(WF_E_INVALID, "y_hat, mean, scale and idx outputs are required");
    if (p->K == 3 && (!out->weight || !out->comp_mean))
        return fail(WF_E_INVALID, "weight and comp_mean outputs are required for K = 3");
    return WF_OK;
}

int wf_decode(wf_plan_t plan, const float* psi, const int32_t* sym, const wf_out* out,
              hipStream_t stream) {
    if (!plan || !psi || !sym) return fail(WF_E_INVALID, "plan, psi or sym is NULL");
    Plan* p = reinterpret_cast<Plan*>(plan);
    int rc = check_out(p, out);
    if (rc != WF_OK) return rc;
    return run_steps(*p, psi, sym, nullptr, nullptr, out, stream);
}

int wf_encode(wf_plan_t plan, const float* psi, const float* y, int32_t* sym_out,
              const wf_out* out, hipStream_t stream) {
    if (!plan || !psi || !y || !sym_out) return fail(WF_E_INVALID, "plan, psi, y or sym_out is NULL");
    Plan* p = reinterpret_cast<Plan*>(plan);
    int rc = check_out(p, out);
    if (rc != WF_OK) return rc;
    return run_steps(*p, psi, nullptr, y, sym_out, out, stream);
}

int wf_plan_sync(wf_plan_t plan, hipStream_t stream) {
    if (!plan) return fail(WF_E_INVALID, "plan is NULL");
    Plan* p = reinterpret_cast<Plan*>(plan);
    WF_HIP(hipStreamSynchronize(stream));
    int err = 0;
    WF_HIP(hipMemcpy(&err, p->d_err, sizeof(int), hipMemcpyDeviceToHost));
    if (err) {
        WF_HIP(hipMemset(p->d_err, 0, sizeof(int)));
        return fail(WF_E_TIMEOUT, "a device-wide wait exceeded its spin budget");
    }
    return WF_OK;
}

void wf_plan_destroy(wf_plan_t plan) { free_plan(reinterpret_cast<Plan*>(plan)); }

}  // extern "C"
