// Internal declarations shared by the host plan code and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "wf.h"

namespace wf {

constexpr int kMaxTaps = 12;
constexpr int kTile = 16;            // MFMA tile edge (rows and columns)
constexpr int kMaxTable = 256;

// Set the calling thread's error message and return `code`.
int fail(int code, const std::string& msg);

// Rows of one wavefront step: B images x n latents each.  Row r belongs to
// image r / n and to grid position order[ptr + r % n].
struct StepRows {
    int n;
    int ptr;
    int nrows;
};

// One batched product of a step: out[r][col] += sum_k A[r][k] * Wt[k][col]
// over the k-range of this launch's z-slice.  A is produced on the fly from
// one of three sources (see ASource).
enum ASource { A_TAPS = 0, A_PSI_CTX = 1, A_HIDDEN = 2 };

struct GemmArgs {
    const float* wp;        // packed weights [Np/16][Kp/16][64 lanes][4]
    int nkb;                // Kp / 16
    int kb_per_split;       // k-blocks per z-slice
    float* out;             // raw fp32 sums [rows][ldo], accumulated atomically
    int ldo;
    const float* y_hat;     // A_TAPS source, NHWC [B][H][W][M]
    const float* psi;       // A_PSI_CTX first half, [B][H][W][2M]
    const float* in;        // dense raw input [rows][ldi] (ctx or hidden sums)
    int ldi;
    const float* in_bias;   // added to `in` on load (padded with zeros)
    float slope;            // LeakyReLU slope applied on load (A_HIDDEN)
    int H, W, M;
    const int* order;       // grid positions of all steps, step-major
    int dy[kMaxTaps], dx[kMaxTaps];
};

struct EpiArgs {
    float* o;               // raw last-layer sums [rows][ldo]; cleared after reading
    int ldo;
    const float* b3;        // [n3]
    const float* table;     // [L]
    int L, M, K, H, W;
    const int* order;
    const int32_t* sym;     // decode input
    const float* y;         // encode input
    int32_t* sym_out;       // encode output
    int encode;
    float *y_hat, *mean, *scale, *weight, *cmean;
    int32_t* idx;
    float* clr[3];          // raw buffers to clear for the next step
    int clr_ld[3];
};

struct Plan {
    // description
    int H, W, M, B, K, d1, d2, n3, mask, precision, driver, L;
    float slope;
    // schedule
    int lambda, T, ntaps;
    int dy[kMaxTaps], dx[kMaxTaps];
    std::vector<int32_t> step_of;        // [H*W]
    std::vector<int> step_ptr, step_n;   // [T]
    int max_rows;
    // padded widths
    int Np1, Np2;                        // d1, d2 rounded up to 16
    // device memory
    int device;
    int* d_order = nullptr;
    float *d_wc = nullptr, *d_w1 = nullptr, *d_w2 = nullptr, *d_w3 = nullptr;
    float *d_bc = nullptr, *d_b1 = nullptr, *d_b2 = nullptr, *d_b3 = nullptr;
    float* d_table = nullptr;
    float *d_ctx = nullptr, *d_h1 = nullptr, *d_h2 = nullptr, *d_o = nullptr;
    int* d_err = nullptr;
};

// Launch every kernel of one decode/encode call on `stream` (per-step driver).
int run_steps(Plan& p, const float* psi, const int32_t* sym, const float* y,
              int32_t* sym_out, const wf_out* out, hipStream_t stream);

}  // namespace wf
