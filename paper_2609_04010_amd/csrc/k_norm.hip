// Time embedding, token/position embedding + first normalisation, and normalisation (LayerNorm or
// RMSNorm, a template parameter of every kernel).
//
// One wavefront per token row; statistics are reduced across the lanes in fp32 from registers.
// LayerNorm: the mean first, then the biased variance of the centred values; y = (x - mean) rstd g + b.
// RMSNorm: the mean square; y = x rstd g, rstd = 1 / sqrt(mean square + eps) (no shift is read).
#include <math.h>

#include "kernels.h"

namespace dd {

// temb_j = sin(tau w_j) (j < d/2), cos(tau w_{j-d/2}) (j >= d/2), w_i = 10000^(-i/(d/2)),
// evaluated in float64 and stored as fp32.
__global__ void temb_kernel(float* temb, int d, double tau) {
    const int j = blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= d) return;
    const int half = d / 2;
    const int i = j < half ? j : j - half;
    const double w = pow(10000.0, -(double)i / (double)half);
    temb[j] = (float)(j < half ? sin(tau * w) : cos(tau * w));
}

dd_status launch_temb(float* temb, int d, double tau, hipStream_t s) {
    ProfScope ps(KC_TEMB, s);
    launch_k(temb_kernel, dim3((d + 255) / 256), dim3(256), 0, s, temb, d, tau);
    return launch_status("time_embedding");
}

template <typename W> DD_DEV float ldw(const W* p, int64_t i);
template <> DD_DEV float ldw<bf16_t>(const bf16_t* p, int64_t i) { return bf16_to_f32(p[i]); }
template <> DD_DEV float ldw<float>(const float* p, int64_t i) { return p[i]; }
template <typename W> DD_DEV void stw(W* p, int64_t i, float v);
template <> DD_DEV void stw<bf16_t>(bf16_t* p, int64_t i, float v) { p[i] = f32_to_bf16(v); }
template <> DD_DEV void stw<float>(float* p, int64_t i, float v) { p[i] = v; }

// NPL = d / 64 elements per lane (d % 64 == 0).
template <typename W, int NPL, bool RMS>
DD_DEV void ln_row(const float (&x)[NPL], int lane, int d, const W* g, const W* b, float eps,
                   W* out) {
    float mean = 0.f;
    if constexpr (!RMS) {
        float s = 0.f;
#pragma unroll
        for (int k = 0; k < NPL; ++k) s += x[k];
        mean = wave_sum(s) / (float)d;
    }
    float q = 0.f;
#pragma unroll
    for (int k = 0; k < NPL; ++k) { const float c = x[k] - mean; q += c * c; }
    const float rstd = 1.0f / sqrtf(wave_sum(q) / (float)d + eps);
#pragma unroll
    for (int k = 0; k < NPL; ++k) {
        const int c = lane + 64 * k;
        if constexpr (RMS) stw<W>(out, c, x[k] * rstd * ldw<W>(g, c));
        else stw<W>(out, c, (x[k] - mean) * rstd * ldw<W>(g, c) + ldw<W>(b, c));
    }
}

template <typename W, int NPL, bool RMS>
__global__ __launch_bounds__(256) void embed_ln_kernel(const int32_t* z, int64_t rows, int L,
                                                       int n_tok, const W* tok, const W* pos,
                                                       const float* temb, const W* g, const W* b,
                                                       float eps, float* h, W* xln, int64_t ldo,
                                                       int32_t* err) {
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= rows) return;
    constexpr int d = NPL * 64;
    int id = z[row];
    if (id < 0 || id >= n_tok) {
        if (lane == 0 && err) atomicOr(err, DD_DEVERR_TOKEN);
        id = id < 0 ? 0 : n_tok - 1;
    }
    const int l = (int)(row % L);
    float x[NPL];
#pragma unroll
    for (int k = 0; k < NPL; ++k) {
        const int c = lane + 64 * k;
        float v = ldw<W>(tok, (int64_t)id * d + c) + ldw<W>(pos, (int64_t)l * d + c);
        if (temb) v += temb[c];
        x[k] = v;
        h[row * d + c] = v;
    }
    ln_row<W, NPL, RMS>(x, lane, d, g, b, eps, xln + row * ldo);
}

template <typename W, int NPL, bool RMS>
__global__ __launch_bounds__(256) void ln_kernel(const float* h, int64_t rows, const W* g,
                                                 const W* b, float eps, W* out, int64_t ldo,
                                                 const int32_t* m_count) {
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (m_count) rows = min(rows, (int64_t)*m_count);
    if (row >= rows) return;
    constexpr int d = NPL * 64;
    float x[NPL];
#pragma unroll
    for (int k = 0; k < NPL; ++k) x[k] = h[row * d + lane + 64 * k];
    ln_row<W, NPL, RMS>(x, lane, d, g, b, eps, out + row * ldo);
}

// Normalisation of one row held as NV groups of four consecutive features per lane (group
// lane + 64 k), written as 8-byte bf16 stores; gg / bb hold the gain and shift of those features
// (bb unused under RMS).  The statistics are wavefront sums by DPP lane moves.
template <int NV, bool RMS>
DD_DEV void ln4_row(const float4 (&x)[NV], int lane, const uint2 (&gg)[NV], const uint2 (&bb)[NV], float eps,
                    bf16_t* out) {
    constexpr int d = NV * 256;
    float mean = 0.f;
    if constexpr (!RMS) {
        float s = 0.f;
#pragma unroll
        for (int k = 0; k < NV; ++k) s += (x[k].x + x[k].y) + (x[k].z + x[k].w);
        mean = wave_sum_dpp(s) / (float)d;
    }
    float q = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const float a0 = x[k].x - mean, a1 = x[k].y - mean, a2 = x[k].z - mean, a3 = x[k].w - mean;
        q += (a0 * a0 + a1 * a1) + (a2 * a2 + a3 * a3);
    }
    const float rstd = 1.0f / sqrtf(wave_sum_dpp(q) / (float)d + eps);
    uint2* orow = (uint2*)out;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int c = lane + 64 * k;
        uint2 o;
        if constexpr (RMS) {
            o.x = pack_bf16x2(x[k].x * rstd * bf16_lo(gg[k].x), x[k].y * rstd * bf16_hi(gg[k].x));
            o.y = pack_bf16x2(x[k].z * rstd * bf16_lo(gg[k].y), x[k].w * rstd * bf16_hi(gg[k].y));
            orow[c] = o;
            continue;
        }
        o.x = pack_bf16x2((x[k].x - mean) * rstd * bf16_lo(gg[k].x) + bf16_lo(bb[k].x),
                          (x[k].y - mean) * rstd * bf16_hi(gg[k].x) + bf16_hi(bb[k].x));
        o.y = pack_bf16x2((x[k].z - mean) * rstd * bf16_lo(gg[k].y) + bf16_lo(bb[k].y),
                          (x[k].w - mean) * rstd * bf16_hi(gg[k].y) + bf16_hi(bb[k].y));
        orow[c] = o;
    }
}

template <int NV, bool RMS>
DD_DEV void load_gain_shift(const bf16_t* g, const bf16_t* b, int lane, uint2 (&gg)[NV], uint2 (&bb)[NV]) {
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        gg[k] = ((const uint2*)g)[lane + 64 * k];
        if constexpr (!RMS) bb[k] = ((const uint2*)b)[lane + 64 * k];
        else bb[k] = make_uint2(0u, 0u);
    }
}

// bf16 output, d % 256 == 0: each lane holds NV = d / 256 groups of four consecutive features,
// read as one 16-byte fp32 load and written as one 8-byte bf16 store.  A wavefront normalises
// LN_RPW consecutive rows and issues the loads of all of them before the first reduction.  Since
// the residual row arrives from the Infinity Cache (the residual projection stores it normally),
// one row per wavefront is the faster choice: 11.7 vs 12.0 us at B16 L1024 d768, 29.7 vs 30.5 us
// at B8 L4096 d1024.
constexpr int LN_RPW = 1;
template <int NV, bool RMS>
__global__ __launch_bounds__(256) void ln_bf16_v4_kernel(const float* h, int64_t rows,
                                                         const bf16_t* g, const bf16_t* b,
                                                         float eps, bf16_t* out, int64_t ldo,
                                                         const int32_t* m_count) {
    const int64_t row0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * LN_RPW;
    const int lane = threadIdx.x & 63;
    if (m_count) rows = min(rows, (int64_t)*m_count);
    if (row0 >= rows) return;
    constexpr int d = NV * 256;
    float4 x[LN_RPW][NV];
#pragma unroll
    for (int r = 0; r < LN_RPW; ++r) {
        if (row0 + r >= rows) break;
        const float4* hr = (const float4*)(h + (row0 + r) * d);
#pragma unroll
        for (int k = 0; k < NV; ++k) x[r][k] = hr[lane + 64 * k];
    }
    uint2 gg[NV], bb[NV];
    load_gain_shift<NV, RMS>(g, b, lane, gg, bb);
#pragma unroll
    for (int r = 0; r < LN_RPW; ++r) {
        if (row0 + r >= rows) break;
        ln4_row<NV, RMS>(x[r], lane, gg, bb, eps, out + (row0 + r) * ldo);
    }
}

// Embedding + first LayerNorm, bf16, d % 256 == 0: token and position rows read four features at a
// time (8-byte loads), the residual row written with 16-byte stores.
template <int NV, bool RMS>
__global__ __launch_bounds__(256) void embed_ln_bf16_v4_kernel(const int32_t* z, int64_t rows, int L,
                                                               int n_tok, const bf16_t* tok,
                                                               const bf16_t* pos, const float* temb,
                                                               const bf16_t* g, const bf16_t* b, float eps,
                                                               float* h, bf16_t* xln, int64_t ldo,
                                                               int32_t* err) {
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= rows) return;
    constexpr int d = NV * 256;
    int id = z[row];
    if (id < 0 || id >= n_tok) {
        if (lane == 0 && err) atomicOr(err, DD_DEVERR_TOKEN);
        id = id < 0 ? 0 : n_tok - 1;
    }
    const int l = (int)(row % L);
    const uint2* tv = (const uint2*)(tok + (int64_t)id * d);
    const uint2* pv = (const uint2*)(pos + (int64_t)l * d);
    float4* hr = (float4*)(h + row * d);
    float4 x[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int c = lane + 64 * k;
        const uint2 a = tv[c], p = pv[c];
        float4 v = make_float4(bf16_lo(a.x) + bf16_lo(p.x), bf16_hi(a.x) + bf16_hi(p.x),
                               bf16_lo(a.y) + bf16_lo(p.y), bf16_hi(a.y) + bf16_hi(p.y));
        if (temb) {
            const float4 t = ((const float4*)temb)[c];
            v.x += t.x; v.y += t.y; v.z += t.z; v.w += t.w;
        }
        x[k] = v;
        hr[c] = v;
    }
    uint2 gg[NV], bb[NV];
    load_gain_shift<NV, RMS>(g, b, lane, gg, bb);
    ln4_row<NV, RMS>(x, lane, gg, bb, eps, xln + row * ldo);
}

#define DD_NPL_CASES(X) X(1) X(2) X(4) X(8) X(12) X(16) X(24) X(32)

template <typename W, bool RMS>
dd_status launch_embed_ln_t(const int32_t* z, int64_t rows, int L, int n_tok, int d, const void* tok,
                            const void* pos, const float* temb, const void* g, const void* b,
                            float eps, float* h, void* xln, int64_t ldo, int32_t* err, hipStream_t s) {
    const dim3 grid((unsigned)ceil_div(rows, 4)), blk(256);
    switch (d / 64) {
#define X(n)                                                                                     \
    case n:                                                                                      \
        launch_k((embed_ln_kernel<W, n, RMS>), grid, blk, 0, s, z, rows, L, n_tok,     \
                           (const W*)tok, (const W*)pos, temb, (const W*)g, (const W*)b, eps, h,  \
                           (W*)xln, ldo, err);                                                   \
        break;
        DD_NPL_CASES(X)
#undef X
        default: set_error("d_model %d unsupported by the normalisation kernels", d); return DD_E_UNSUPPORTED;
    }
    return launch_status("embed_ln");
}

template <bool RMS>
void launch_embed_ln_v4(int d, dim3 grid, const int32_t* z, int64_t rows, int L, int n_tok,
                        const bf16_t* tk, const bf16_t* ps, const float* temb, const bf16_t* g,
                        const bf16_t* b, float eps, float* h, bf16_t* o, int64_t ldo, int32_t* err,
                        hipStream_t s) {
    const dim3 blk(256);
    if (d == 768)
        launch_k((embed_ln_bf16_v4_kernel<3, RMS>), grid, blk, 0, s, z, rows, L, n_tok, tk, ps, temb, g, b, eps, h, o, ldo, err);
    else if (d == 1024)
        launch_k((embed_ln_bf16_v4_kernel<4, RMS>), grid, blk, 0, s, z, rows, L, n_tok, tk, ps, temb, g, b, eps, h, o, ldo, err);
    else
        launch_k((embed_ln_bf16_v4_kernel<8, RMS>), grid, blk, 0, s, z, rows, L, n_tok, tk, ps, temb, g, b, eps, h, o, ldo, err);
}

dd_status launch_embed_ln(int dtype, int norm, const int32_t* z, int64_t rows, int L, int n_tok, int d,
                          const void* tok, const void* pos, const float* temb, const void* g,
                          const void* b, float eps, float* h, void* xln, int64_t ldo, int32_t* err,
                          hipStream_t s) {
    const bool rms = norm == DD_NORM_RMS;
    ProfScope ps(KC_EMBED_LN, s);
    if (dtype == DD_BF16 && (d == 768 || d == 1024 || d == 2048) && ldo % 4 == 0) {
        const dim3 grid((unsigned)ceil_div(rows, 4));
        const bf16_t *tk = (const bf16_t*)tok, *ps_ = (const bf16_t*)pos, *gg = (const bf16_t*)g, *bb = (const bf16_t*)b;
        bf16_t* o = (bf16_t*)xln;
        if (rms) launch_embed_ln_v4<true>(d, grid, z, rows, L, n_tok, tk, ps_, temb, gg, bb, eps, h, o, ldo, err, s);
        else launch_embed_ln_v4<false>(d, grid, z, rows, L, n_tok, tk, ps_, temb, gg, bb, eps, h, o, ldo, err, s);
        return launch_status("embed_ln");
    }
    if (dtype == DD_BF16)
        return rms ? launch_embed_ln_t<bf16_t, true>(z, rows, L, n_tok, d, tok, pos, temb, g, b, eps, h, xln, ldo, err, s)
                   : launch_embed_ln_t<bf16_t, false>(z, rows, L, n_tok, d, tok, pos, temb, g, b, eps, h, xln, ldo, err, s);
    return rms ? launch_embed_ln_t<float, true>(z, rows, L, n_tok, d, tok, pos, temb, g, b, eps, h, xln, ldo, err, s)
               : launch_embed_ln_t<float, false>(z, rows, L, n_tok, d, tok, pos, temb, g, b, eps, h, xln, ldo, err, s);
}

template <typename W, bool RMS>
dd_status launch_ln_t(const float* h, int64_t rows, int d, const void* g, const void* b, float eps,
                      void* out, int64_t ldo, hipStream_t s, const int32_t* m_count) {
    const dim3 grid((unsigned)ceil_div(rows, 4)), blk(256);
    switch (d / 64) {
#define X(n)                                                                                     \
    case n:                                                                                      \
        launch_k((ln_kernel<W, n, RMS>), grid, blk, 0, s, h, rows, (const W*)g,       \
                           (const W*)b, eps, (W*)out, ldo, m_count);                             \
        break;
        DD_NPL_CASES(X)
#undef X
        default: set_error("d_model %d unsupported by the normalisation kernels", d); return DD_E_UNSUPPORTED;
    }
    return launch_status("layernorm");
}

template <bool RMS>
void launch_ln_v4(int d, dim3 grid, const float* h, int64_t rows, const bf16_t* g, const bf16_t* b,
                  float eps, bf16_t* o, int64_t ldo, hipStream_t s, const int32_t* mc) {
    const dim3 blk(256);
    if (d == 768) launch_k((ln_bf16_v4_kernel<3, RMS>), grid, blk, 0, s, h, rows, g, b, eps, o, ldo, mc);
    else if (d == 1024) launch_k((ln_bf16_v4_kernel<4, RMS>), grid, blk, 0, s, h, rows, g, b, eps, o, ldo, mc);
    else launch_k((ln_bf16_v4_kernel<8, RMS>), grid, blk, 0, s, h, rows, g, b, eps, o, ldo, mc);
}

dd_status launch_ln(int dtype, int norm, const float* h, int64_t rows, int d, const void* g, const void* b,
                    float eps, void* out, int64_t ldo, hipStream_t s, const int32_t* m_count) {
    const bool rms = norm == DD_NORM_RMS;
    ProfScope ps(KC_LN, s);
    if (dtype == DD_BF16 && (d == 768 || d == 1024 || d == 2048) && ldo % 4 == 0) {
        const dim3 grid((unsigned)ceil_div(rows, 4 * LN_RPW));
        const bf16_t* gg = (const bf16_t*)g;
        const bf16_t* bb = (const bf16_t*)b;
        bf16_t* o = (bf16_t*)out;
        if (rms) launch_ln_v4<true>(d, grid, h, rows, gg, bb, eps, o, ldo, s, m_count);
        else launch_ln_v4<false>(d, grid, h, rows, gg, bb, eps, o, ldo, s, m_count);
        return launch_status("layernorm");
    }
    if (dtype == DD_BF16)
        return rms ? launch_ln_t<bf16_t, true>(h, rows, d, g, b, eps, out, ldo, s, m_count)
                   : launch_ln_t<bf16_t, false>(h, rows, d, g, b, eps, out, ldo, s, m_count);
    return rms ? launch_ln_t<float, true>(h, rows, d, g, b, eps, out, ldo, s, m_count)
               : launch_ln_t<float, false>(h, rows, d, g, b, eps, out, ldo, s, m_count);
}

bool ln_supported(int d) {
    switch (d / 64) {
#define X(n) case n:
        DD_NPL_CASES(X)
#undef X
        return d % 64 == 0;
        default: return false;
    }
}

}  // namespace dd
