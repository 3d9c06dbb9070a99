// Philox4x32-10 counter-based generator and the transforms of one 32-bit word
// into the sampler's noise (device code).
//
// Philox4x32 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as
// 1, 2, 3", SC'11, sec. 4.2): each of 10 rounds multiplies counter words 0 and
// 2 by odd 32-bit constants, feeds the high halves xored with the other counter
// words and the key into words 0 and 2, the low halves into words 1 and 3, and
// advances the key by the Weyl constants.
//
// Word -> noise (this library's definition, exact in float64):
//   u = (w + 1/2) 2^-32,  c = 1 - u = (2^32 - 1 - w + 1/2) 2^-32
//   E = -log u  (as -log1p(-c) when u >= 1/2),  Gumbel G = -log E
//   normal N = Phi^-1(u)  (as -Phi^-1(c) when u >= 1/2)
#pragma once

#include "common.h"

namespace dd {

enum Stream : uint32_t { STREAM_TOP = 0, STREAM_CLASS = 1, STREAM_LATENT = 2, STREAM_PARAM = 3, STREAM_VERIFY = 4,
                         STREAM_GROUP_U = 5 };

struct Words4 {
    uint32_t w[4];
};

DD_DEV Words4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                            uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c0;
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)c2;
        const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
        const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
        c1 = (uint32_t)p1;
        c3 = (uint32_t)p0;
        c0 = n0;
        c2 = n2;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    Words4 o;
    o.w[0] = c0; o.w[1] = c1; o.w[2] = c2; o.w[3] = c3;
    return o;
}

// Word for (stream, step, row, index): counter (index >> 2, row, step, stream), word index & 3.
DD_DEV uint32_t counter_word(uint64_t seed, uint32_t stream, uint32_t step, uint32_t row,
                             uint32_t index) {
    const Words4 b = philox4x32_10(index >> 2, row, step, stream, (uint32_t)seed,
                                   (uint32_t)(seed >> 32));
    // selects, not an indexed load: a runtime index into the array would put it in scratch memory
    const uint32_t i = index & 3u;
    return i == 0 ? b.w[0] : i == 1 ? b.w[1] : i == 2 ? b.w[2] : b.w[3];
}

DD_DEV double word_exponential(uint32_t w) {
    if (w >= 0x80000000u) {
        const double c = ((double)(0xFFFFFFFFu - w) + 0.5) * 0x1p-32;
        return -log1p(-c);
    }
    return -log(((double)w + 0.5) * 0x1p-32);
}

DD_DEV double word_gumbel(uint32_t w) { return -log(word_exponential(w)); }

// The same transforms in fp32 (relative error of E about 2^-23, so G is within ~1e-7 of the
// float64 value); the complement c = 1 - u keeps E accurate as u -> 1.
DD_DEV float word_gumbel_f(uint32_t w) {
    float e;
    if (w >= 0x80000000u) e = -log1pf(-(((float)(0xFFFFFFFFu - w) + 0.5f) * 0x1p-32f));
    else e = -logf(((float)w + 0.5f) * 0x1p-32f);
    return -logf(e);
}

DD_DEV double word_normal(uint32_t w) {
    if (w >= 0x80000000u) return -normcdfinv(((double)(0xFFFFFFFFu - w) + 0.5) * 0x1p-32);
    return normcdfinv(((double)w + 0.5) * 0x1p-32);
}

}  // namespace dd
