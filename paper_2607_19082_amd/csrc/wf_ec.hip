// Entropy coding of the symbols with rANS: the plan's frequency tables, the
// decoder states of a decode from streams, and the stream encoder that runs
// after an encode.
//
// The entropy model is the mean-scale Gaussian of the context model
// (Sec. II-A): a symbol s = y - mean (rounded) is coded with the discretised
// zero-mean Gaussian of its scale level l, whose scale is the level's table
// value T_l.  The paper pairs the wavefront decode with rANS (Sec. III-C);
// here every (image, grid row, channel) has a stream of its own, holding the
// row's symbols in column order, so a wavefront step decodes at most one
// symbol of each stream and the decode runs inside the step loop on the GPU.
//
// Tables, per level l: support n_l = max(1, ceil(6 T_l)); symbols u = s + n_l
// for |s| <= n_l and an escape u = 2 n_l + 1; with r = T_l sqrt 2,
// a = (|s| - 1/2) / r and b = (|s| + 1/2) / r the masses are p(0) = 1 - erfc(b),
// p(s) = (erfc(a) - erfc(b)) / 2 and p(escape) = erfc((n_l + 1/2) / r); the
// frequencies are f_u = 1 + floor(p_u (2^16 - (2 n_l + 2))) with the rest of
// 2^16 added to s = 0.  An escaped symbol is followed by e = 2(|s| - n_l - 1)
// + (s < 0) in 15-bit chunks, low first, each a uniform 16-bit value whose
// top bit marks another chunk.
//
// The 3-component mixture (K = 3) codes each symbol with the mixture of its
// channel's components around the mixture mean; its per-latent frequencies
// come from quantised parameters and the per-level integer CDFs built here
// (mix_tables; the arithmetic is with the decode, next to mix_param).
//
// Coder: state x in [2^31, 2^63), 32-bit renormalisation words.  Encoding a
// symbol of frequency f and cumulative frequency c emits the low word of x
// (x >>= 32) when x >= f 2^47, then x = floor(x / f) 2^16 + (x mod f) + c;
// decoding inverts it.  A stream is the final state (high word, low word)
// followed by the emitted words in reverse order of emission.
#include <algorithm>
#include <cmath>
#include <vector>

#include "wf_device.h"

namespace wf {

constexpr int kEcTailSigmas = 6;
constexpr int kEcMaxEscapeWords = 3;   // chunks of a 32-bit excess

// ---- tables (host) -------------------------------------------------------

static int support_of(float t) {
    const double n = std::ceil((double)kEcTailSigmas * (double)t);
    return n < 1.0 ? 1 : (n > (double)kEcMaxSupport + 1 ? kEcMaxSupport + 1 : (int)n);
}

static double level_mass(int u, int n, double sigma) {
    const double r = sigma * std::sqrt(2.0);
    if (u == 2 * n + 1) return std::erfc(((double)n + 0.5) / r);
    const int s = u > n ? u - n : n - u;
    const double b = ((double)s + 0.5) / r;
    if (s == 0) return 1.0 - std::erfc(b);
    const double a = ((double)s - 0.5) / r;
    return 0.5 * (std::erfc(a) - std::erfc(b));
}

// Frequency tables of a scale table: n [L], base [L+1] (first cumulative
// entry of each level), cum (2n+3 entries per level) and, when lut != NULL,
// for every 16-slot bucket [L][kEcLut] the symbol u holding its first slot
// with cum[u] and cum[u + 1], packed as u | cum[u] << 16 | cum[u + 1] << 32.
static int ec_tables(const float* table, int L, std::vector<int32_t>& n, std::vector<int64_t>& base,
                     std::vector<uint32_t>& cum, std::vector<uint64_t>* lut) {
    n.assign(L, 0);
    base.assign(L + 1, 0);
    for (int l = 0; l < L; ++l) {
        n[l] = support_of(table[l]);
        if (n[l] > kEcMaxSupport) return fail(WF_E_UNSUPPORTED, "entropy coding: a scale level is too wide");
        base[l + 1] = base[l] + 2 * (int64_t)n[l] + 3;
    }
    cum.assign((size_t)base[L], 0u);
    if (lut) lut->assign((size_t)L * kEcLut, 0);
    std::vector<uint32_t> f;
    for (int l = 0; l < L; ++l) {
        const int K = 2 * n[l] + 2;
        const double spread = (double)((1u << kEcPrecBits) - (uint32_t)K);
        f.assign(K, 0u);
        uint32_t sum = 0;
        for (int u = 0; u < K; ++u) {
            f[u] = 1u + (uint32_t)std::floor(level_mass(u, n[l], (double)table[l]) * spread);
            sum += f[u];
        }
        f[n[l]] += (1u << kEcPrecBits) - sum;
        uint32_t* c = cum.data() + base[l];
        for (int u = 0; u < K; ++u) c[u + 1] = c[u] + f[u];
        if (lut) {
            uint64_t* q = lut->data() + (size_t)l * kEcLut;
            int u = 0;
            for (int b = 0; b < kEcLut; ++b) {
                const uint32_t slot = (uint32_t)b << kEcLutShift;
                while (c[u + 1] <= slot) ++u;
                q[b] = (uint64_t)u | ((uint64_t)c[u] << 16) | ((uint64_t)c[u + 1] << 32);
            }
        }
    }
    return WF_OK;
}

// The mixture coder's level tables (K = 3): X_l = 16 (n_l + 1) and the
// integer CDF on sixteenths of a symbol, G_l(x) = floor(2^20 Phi(x / (16 T_l))
// + 1/2) for x = -X_l..X_l (Phi(z) = erfc(-z / sqrt 2) / 2), level after level.
static int mix_tables(const float* table, int L, std::vector<int32_t>& X, std::vector<int64_t>& base,
                      std::vector<uint32_t>& G) {
    X.assign(L, 0);
    base.assign(L + 1, 0);
    for (int l = 0; l < L; ++l) {
        const int n = support_of(table[l]);
        if (n > kEcMaxSupport) return fail(WF_E_UNSUPPORTED, "entropy coding: a scale level is too wide");
        X[l] = kMixFine * (n + 1);
        base[l + 1] = base[l] + 2 * (int64_t)X[l] + 1;
    }
    G.assign((size_t)base[L], 0u);
    for (int l = 0; l < L; ++l) {
        const double r = kMixFine * (double)table[l] * std::sqrt(2.0);
        uint32_t* g = G.data() + base[l];
        for (int x = -X[l]; x <= X[l]; ++x) {
            const double phi = 0.5 * std::erfc(-(double)x / r);
            g[x + X[l]] = (uint32_t)std::floor(phi * (double)(1u << kMixCdfBits) + 0.5);
        }
    }
    return WF_OK;
}

template <class T>
static int ec_alloc(Plan* p, T** dst, size_t count) {
    hipError_t e = hipMalloc((void**)dst, count * sizeof(T));
    if (e != hipSuccess) return fail(WF_E_NOMEM, std::string("entropy coder workspace: ") + hipGetErrorString(e));
    p->owned.push_back((void*)*dst);
    return WF_OK;
}
template <class T>
static int ec_upload(Plan* p, T** dst, const std::vector<T>& v) {
    int rc = ec_alloc(p, dst, v.size());
    if (rc != WF_OK) return rc;
    hipError_t e = hipMemcpy(*dst, v.data(), v.size() * sizeof(T), hipMemcpyHostToDevice);
    if (e != hipSuccess) return fail(WF_E_HIP, std::string("entropy coder tables: ") + hipGetErrorString(e));
    return WF_OK;
}

int build_ec(Plan* p, const float* scale_table, int L) {
    int rc;
    if (p->K == 1) {
        std::vector<int32_t> n;
        std::vector<int64_t> base;
        std::vector<uint32_t> cum;
        std::vector<uint64_t> lut;
        if ((rc = ec_tables(scale_table, L, n, base, cum, &lut)) != WF_OK) return rc;
        std::vector<int32_t> base32(L);
        for (int l = 0; l < L; ++l) base32[l] = (int32_t)base[l];
        if ((rc = ec_upload(p, &p->ec_n, n)) != WF_OK || (rc = ec_upload(p, &p->ec_base, base32)) != WF_OK ||
            (rc = ec_upload(p, &p->ec_cum, cum)) != WF_OK || (rc = ec_upload(p, &p->ec_lut, lut)) != WF_OK)
            return rc;
    } else {
        std::vector<int32_t> X;
        std::vector<int64_t> base;
        std::vector<uint32_t> G;
        if ((rc = mix_tables(scale_table, L, X, base, G)) != WF_OK) return rc;
        // every latent's coded symbols must number at most kMixMaxSymbols
        const int Xmax = *std::max_element(X.begin(), X.end());
        if ((2 * (int64_t)kMixQmax + 2 * (int64_t)Xmax) / kMixFine + 2 > kMixMaxSymbols)
            return fail(WF_E_UNSUPPORTED, "entropy coding: the scale table is too wide for the mixture coder");
        if (base[L] >= (int64_t)1 << 31) return fail(WF_E_UNSUPPORTED, "entropy coding: mixture tables too large");
        std::vector<int32_t> base32(L);
        for (int l = 0; l < L; ++l) base32[l] = (int32_t)base[l];
        if ((rc = ec_upload(p, &p->mix_X, X)) != WF_OK || (rc = ec_upload(p, &p->mix_base, base32)) != WF_OK ||
            (rc = ec_upload(p, &p->mix_G, G)) != WF_OK)
            return rc;
    }
    const size_t ns = (size_t)p->B * p->H * p->M;
    const size_t per = 2 + (size_t)(1 + kEcMaxEscapeWords) * p->W;   // words one stream can take
    if ((rc = ec_alloc(p, &p->ec_x, ns)) != WF_OK || (rc = ec_alloc(p, &p->ec_pos, ns)) != WF_OK ||
        (rc = ec_alloc(p, &p->ec_end, ns)) != WF_OK || (rc = ec_alloc(p, &p->ec_len, ns)) != WF_OK ||
        (rc = ec_alloc(p, &p->ec_words, ns * per)) != WF_OK)
        return rc;
    p->ec = 1;
    return WF_OK;
}

// ---- decode from streams: per-stream start --------------------------------

// Stream k starts at offsets[k] and ends at offsets[k + 1], both clamped to
// the caller's n_words; its first two words are the state.  A stream too
// short, out of order or with a state below 2^31 records a stream error.
__global__ void k_ec_init(const uint32_t* __restrict__ bits, long long n_words, const uint32_t* __restrict__ offs,
                          int ns, uint64_t* __restrict__ ex, uint32_t* __restrict__ epos, uint32_t* __restrict__ eend,
                          int* err) {
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= ns) return;
    const long long lim = n_words < 0xffffffffLL ? n_words : 0xffffffffLL;
    const long long b0 = offs[k], b1 = offs[k + 1];
    const long long beg = b0 < lim ? b0 : lim, end = b1 < lim ? b1 : lim;
    bool bad = end < beg + 2 || b1 > lim;
    uint64_t x = 0;
    if (!bad) x = ((uint64_t)bits[beg] << 32) | bits[beg + 1];
    bad |= x < (1ull << 31);
    ex[k] = bad ? (1ull << 31) : x;
    epos[k] = (uint32_t)(bad ? end : beg + 2);
    eend[k] = (uint32_t)end;
    if (bad) __hip_atomic_store(err, kErrStream, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

int enqueue_ec_init(Plan& p, const uint32_t* bits, int64_t n_words, const uint32_t* offsets, hipStream_t stream) {
    const int ns = p.B * p.H * p.M;
    hipLaunchKernelGGL(k_ec_init, dim3((ns + 255) / 256), dim3(256), 0, stream, bits, (long long)n_words, offsets, ns,
                       p.ec_x, p.ec_pos, p.ec_end, p.d_err);
    return WF_OK;
}

// ---- stream encoder ---------------------------------------------------------

__device__ __forceinline__ void ec_push(uint64_t& x, uint32_t c, uint32_t f, uint32_t* __restrict__ w, uint32_t& n) {
    if (x >= ((uint64_t)f << 47)) {
        w[n++] = (uint32_t)x;
        x >>= 32;
    }
    x = ((x / f) << kEcPrecBits) + (x % f) + c;
}

// One thread per stream (image b, grid row i, channel c): the row's symbols
// from the last column to the first, at the scale levels of the encode; the
// emitted words go to the stream's scratch slot in emission order.
__global__ void k_ec_encode(const int32_t* __restrict__ sym, const int32_t* __restrict__ idx, int H, int W, int M,
                            int ns, int L, const int32_t* __restrict__ tn, const int32_t* __restrict__ tbase,
                            const uint32_t* __restrict__ tcum, uint32_t* __restrict__ words, int per,
                            uint64_t* __restrict__ xs, uint32_t* __restrict__ len, int* err) {
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= ns) return;
    const int c = k % M, row = k / M;   // row = b * H + i
    uint32_t* w = words + (size_t)k * per;
    uint64_t x = 1ull << 31;
    uint32_t n = 0;
    bool bad = false;
    for (int j = W - 1; j >= 0; --j) {
        const size_t q = ((size_t)row * W + j) * M + c;
        const int lvl = idx[q];
        const int32_t s = sym[q];
        if (lvl < 0 || lvl >= L) {
            bad = true;
            break;
        }
        const int sn = tn[lvl];
        const uint32_t* cum = tcum + tbase[lvl];
        int u;
        if (s >= -sn && s <= sn) {
            u = s + sn;
        } else {
            u = 2 * sn + 1;
            const int64_t mag = s < 0 ? -(int64_t)s : (int64_t)s;
            const uint64_t e = 2u * (uint64_t)(mag - sn - 1) + (s < 0 ? 1u : 0u);
            int nc = 1;
            while (nc < kEcMaxEscapeWords && (e >> (15 * nc))) ++nc;
            for (int q2 = nc - 1; q2 >= 0; --q2) {
                const uint32_t ch = (uint32_t)((e >> (15 * q2)) & 0x7fffu) | (q2 < nc - 1 ? 0x8000u : 0u);
                ec_push(x, ch, 1u, w, n);
            }
        }
        ec_push(x, cum[u], cum[u + 1] - cum[u], w, n);
    }
    xs[k] = x;
    len[k] = n;
    if (bad) __hip_atomic_store(err, kErrStream, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The same for the 3-component mixture: each symbol's frequencies from the
// encode's weights, component means, mixture mean and scale levels.
__global__ void k_ec_encode_mix(const int32_t* __restrict__ sym, const float* __restrict__ weight,
                                const float* __restrict__ cmean, const float* __restrict__ mean,
                                const int32_t* __restrict__ idx, int H, int W, int M, int ns, int L,
                                const int32_t* __restrict__ tX, const int32_t* __restrict__ tbase,
                                const uint32_t* __restrict__ tG, uint32_t* __restrict__ words, int per,
                                uint64_t* __restrict__ xs, uint32_t* __restrict__ len, int* err) {
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= ns) return;
    CallPtrs t{};
    t.mix_X = tX;
    t.mix_base = tbase;
    t.mix_G = tG;
    const int c = k % M, row = k / M;   // row = b * H + i
    uint32_t* w = words + (size_t)k * per;
    uint64_t x = 1ull << 31;
    uint32_t n = 0;
    bool bad = false;
    for (int j = W - 1; j >= 0; --j) {
        const size_t lat = (size_t)row * W + j;
        float w3[3], m3[3];
        int l3[3];
#pragma unroll
        for (int kk = 0; kk < 3; ++kk) {
            const size_t q = (lat * 3 + kk) * M + c;
            w3[kk] = weight[q];
            m3[kk] = cmean[q];
            l3[kk] = idx[q];
            bad |= l3[kk] < 0 || l3[kk] >= L;
        }
        if (bad) break;
        const MixParam p = mix_param(&t, w3, m3, mean[lat * M + c], l3);
        if (p.hi - p.lo + 1 > kMixMaxSymbols) {
            bad = true;
            break;
        }
        const int32_t s = sym[lat * M + c];
        if (s >= p.lo && s <= p.hi) {
            const uint32_t c0 = mix_cum(&t, p, s), c1 = mix_cum(&t, p, s + 1);
            ec_push(x, c0, c1 - c0, w, n);
            continue;
        }
        const uint64_t e = s < p.lo ? 2u * (uint64_t)((int64_t)p.lo - 1 - s) + 1u
                                    : 2u * (uint64_t)((int64_t)s - p.hi - 1);
        int nc = 1;
        while (nc < kEcMaxEscapeWords && (e >> (15 * nc))) ++nc;
        for (int q2 = nc - 1; q2 >= 0; --q2) {
            const uint32_t ch = (uint32_t)((e >> (15 * q2)) & 0x7fffu) | (q2 < nc - 1 ? 0x8000u : 0u);
            ec_push(x, ch, 1u, w, n);
        }
        ec_push(x, (1u << kEcPrecBits) - 1u, 1u, w, n);
    }
    xs[k] = x;
    len[k] = n;
    if (bad) __hip_atomic_store(err, kErrStream, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Offsets of the streams (exclusive prefix sum of 2 + emitted words) in one
// workgroup; offsets[ns] is the total.  A total above the caller's capacity
// records a capacity error (the streams are then not written).
constexpr int kScanThreads = 1024;
__global__ __launch_bounds__(kScanThreads) void k_ec_scan(const uint32_t* __restrict__ len, int ns,
                                                          uint32_t* __restrict__ offs, long long cap, int* err) {
    __shared__ unsigned long long part[kScanThreads];
    const int t = threadIdx.x;
    const int chunk = (ns + kScanThreads - 1) / kScanThreads;
    const int k0 = min(ns, t * chunk), k1 = min(ns, k0 + chunk);
    unsigned long long sum = 0;
    for (int k = k0; k < k1; ++k) sum += 2ull + len[k];
    part[t] = sum;
    __syncthreads();
    for (int d = 1; d < kScanThreads; d <<= 1) {   // inclusive scan (Hillis-Steele)
        const unsigned long long v = t >= d ? part[t - d] : 0ull;
        __syncthreads();
        part[t] += v;
        __syncthreads();
    }
    unsigned long long run = part[t] - sum;
    const unsigned long long total = part[kScanThreads - 1];
    const bool over = total > (unsigned long long)cap || total > 0xffffffffull;
    for (int k = k0; k < k1; ++k) {
        offs[k] = (uint32_t)run;
        run += 2ull + len[k];
    }
    if (t == 0) {
        offs[ns] = (uint32_t)(total > 0xffffffffull ? 0xffffffffull : total);
        if (over) __hip_atomic_store(err, kErrCapacity, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// Stream k into the caller's buffer: the state, then the emitted words in
// reverse order of emission.
__global__ void k_ec_compact(const uint32_t* __restrict__ words, int per, const uint64_t* __restrict__ xs,
                             const uint32_t* __restrict__ len, const uint32_t* __restrict__ offs, int ns,
                             long long cap, uint32_t* __restrict__ bits) {
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= ns) return;
    const unsigned long long total = offs[ns];
    if (total > (unsigned long long)cap) return;
    const uint32_t o = offs[k], n = len[k];
    const uint32_t* w = words + (size_t)k * per;
    bits[o] = (uint32_t)(xs[k] >> 32);
    bits[o + 1] = (uint32_t)xs[k];
    for (uint32_t q = 0; q < n; ++q) bits[o + 2 + q] = w[n - 1 - q];
}

int enqueue_ec_encode(Plan& p, const int32_t* sym, const wf_out& out, uint32_t* bits, int64_t cap, uint32_t* offsets,
                      hipStream_t stream) {
    const int ns = p.B * p.H * p.M;
    const int per = 2 + (1 + kEcMaxEscapeWords) * p.W;
    const dim3 g((ns + 255) / 256), b(256);
    if (p.K == 1)
        hipLaunchKernelGGL(k_ec_encode, g, b, 0, stream, sym, out.idx, p.H, p.W, p.M, ns, p.L, p.ec_n, p.ec_base,
                           p.ec_cum, p.ec_words, per, p.ec_x, p.ec_len, p.d_err);
    else
        hipLaunchKernelGGL(k_ec_encode_mix, g, b, 0, stream, sym, out.weight, out.comp_mean, out.mean, out.idx, p.H,
                           p.W, p.M, ns, p.L, p.mix_X, p.mix_base, p.mix_G, p.ec_words, per, p.ec_x, p.ec_len,
                           p.d_err);
    hipLaunchKernelGGL(k_ec_scan, dim3(1), dim3(kScanThreads), 0, stream, p.ec_len, ns, offsets, (long long)cap,
                       p.d_err);
    hipLaunchKernelGGL(k_ec_compact, g, b, 0, stream, p.ec_words, per, p.ec_x, p.ec_len, offsets, ns, (long long)cap,
                       bits);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(WF_E_HIP, std::string("entropy coder launch: ") + hipGetErrorString(e));
    return WF_OK;
}

}  // namespace wf

using namespace wf;

extern "C" int wf_ec_tables(const float* scale_table, int32_t L, int32_t* n_out, int64_t* base_out, uint32_t* cum,
                            int64_t cum_cap) {
    if (!scale_table || L < 2 || L > kMaxTable) return fail(WF_E_INVALID, "scale table pointer or length");
    std::vector<int32_t> n;
    std::vector<int64_t> base;
    std::vector<uint32_t> c;
    const int rc = ec_tables(scale_table, L, n, base, c, nullptr);
    if (rc != WF_OK) return rc;
    if (n_out) std::copy(n.begin(), n.end(), n_out);
    if (base_out) std::copy(base.begin(), base.end(), base_out);
    if (cum) {
        if (cum_cap < base[L]) return fail(WF_E_INVALID, "cum holds fewer entries than the tables");
        std::copy(c.begin(), c.end(), cum);
    }
    return WF_OK;
}

extern "C" int wf_mix_tables(const float* scale_table, int32_t L, int32_t* X_out, int64_t* base_out, uint32_t* G,
                             int64_t G_cap) {
    if (!scale_table || L < 2 || L > kMaxTable) return fail(WF_E_INVALID, "scale table pointer or length");
    std::vector<int32_t> X;
    std::vector<int64_t> base;
    std::vector<uint32_t> g;
    const int rc = mix_tables(scale_table, L, X, base, g);
    if (rc != WF_OK) return rc;
    if (X_out) std::copy(X.begin(), X.end(), X_out);
    if (base_out) std::copy(base.begin(), base.end(), base_out);
    if (G) {
        if (G_cap < base[L]) return fail(WF_E_INVALID, "G holds fewer entries than the tables");
        std::copy(g.begin(), g.end(), G);
    }
    return WF_OK;
}
