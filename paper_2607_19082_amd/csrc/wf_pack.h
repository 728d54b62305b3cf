// Host-side packing of weight panels into the MFMA operand order of the
// kernels (fp32 k-blocks of 16, bf16 k-blocks of 32), shared by the plans of
// the step loop and of the transforms.
#pragma once

#include <cstdint>
#include <cstring>
#include <vector>

#include "wf_internal.h"

namespace wf {

// Pack Wt[k][n] (k < K, n < N; zero up to the padded sizes Kp, Np the
// kernels use) into the MFMA operand order of the step kernels: for column
// tile ct and k-block kb (16 values of k), lane l holds
// Wt[kb*16 + (l/16)*4 + q][ct*16 + l%16] for q = 0..3.
template <class F>
inline std::vector<float> pack_panel(int K, int N, int Kp, int Np, F wt) {
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

// bf16 bits of v, round to nearest even (finite inputs).
inline uint16_t bf16_round(float v) {
    uint32_t u;
    std::memcpy(&u, &v, 4);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// v rounded to bf16, as an fp32 value.
inline float bf16_value_of(float v) {
    const uint32_t u = (uint32_t)bf16_round(v) << 16;
    float r;
    std::memcpy(&r, &u, 4);
    return r;
}

// The same for bf16 operands, k-blocks of 32: lane l holds
// Wt[kb*32 + (l/16)*8 + q][ct*16 + l%16] for q = 0..7, rounded to bf16.
template <class F>
inline std::vector<uint16_t> pack_panel_bf16(int K, int N, int Kp, int Np, F wt) {
    const int nkb = Kp / 32;
    std::vector<uint16_t> out((size_t)Np * Kp, 0);
    for (int ct = 0; ct < Np / kTile; ++ct)
        for (int kb = 0; kb < nkb; ++kb)
            for (int l = 0; l < 64; ++l)
                for (int q = 0; q < 8; ++q) {
                    int k = kb * 32 + (l / 16) * 8 + q;
                    int n = ct * kTile + l % 16;
                    float v = (k < K && n < N) ? wt(k, n) : 0.0f;
                    out[(((size_t)ct * nkb + kb) * 64 + l) * 8 + q] = bf16_round(v);
                }
    return out;
}

}  // namespace wf
