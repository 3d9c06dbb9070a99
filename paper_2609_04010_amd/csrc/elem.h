// Logit rows as 16-byte chunks: element access for bf16 (8 per chunk) and fp32 (4 per chunk) rows,
// -inf fill and clipping of the ragged last chunk (device code).
#pragma once

#include "common.h"

namespace dd {

constexpr float LOG2E = 1.4426950408889634f;

template <typename T> struct Elem;
template <> struct Elem<bf16_t> {
    static constexpr int E = 8;  // elements per 16-byte chunk
    static constexpr uint4 NEG_INF4 = {0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u};
    // elements n.. of the chunk become -inf (0 < n < E)
    DD_DEV static void clip(uint4& c, int n) {
        uint32_t w[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint32_t hi_cut = (w[k] & 0xFFFFu) | 0xFF800000u;
            w[k] = (2 * k + 1 < n) ? w[k] : (2 * k < n) ? hi_cut : 0xFF80FF80u;
        }
        c = make_uint4(w[0], w[1], w[2], w[3]);
    }
    DD_DEV static float get(const uint4& c, int e) {
        const uint32_t w = (e < 2) ? c.x : (e < 4) ? c.y : (e < 6) ? c.z : c.w;
        return (e & 1) ? bf16_hi(w) : bf16_lo(w);
    }
    DD_DEV static float load1(const void* p, int64_t i) { return bf16_to_f32(((const bf16_t*)p)[i]); }
};
template <> struct Elem<float> {
    static constexpr int E = 4;
    static constexpr uint4 NEG_INF4 = {0xFF800000u, 0xFF800000u, 0xFF800000u, 0xFF800000u};
    DD_DEV static void clip(uint4& c, int n) {
        uint32_t w[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) w[k] = (k < n) ? w[k] : 0xFF800000u;
        c = make_uint4(w[0], w[1], w[2], w[3]);
    }
    DD_DEV static float get(const uint4& c, int e) {
        const uint32_t w = (e == 0) ? c.x : (e == 1) ? c.y : (e == 2) ? c.z : c.w;
        return __uint_as_float(w);
    }
    DD_DEV static float load1(const void* p, int64_t i) { return ((const float*)p)[i]; }
};

}  // namespace dd
