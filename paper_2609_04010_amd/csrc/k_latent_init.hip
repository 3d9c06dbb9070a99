// Gaussian-latent argmax (App. A.5) and seeded parameter initialisation.
#include <math.h>

#include "kernels.h"
#include "rng.h"

namespace dd {

// z = argmax_v (alpha_tilde [v == x] + sigma eps_v), eps_v = Phi^-1(u_v).
// Phi^-1 is increasing, so among v != x the largest latent belongs to the largest
// word; only two normals per row are evaluated (in float64).  Ties (equal words or
// equal scores) go to the lowest index.
__global__ __launch_bounds__(256) void latent_kernel(const int32_t* x, int32_t V, double at,
                                                     double sigma, uint64_t seed, uint32_t step,
                                                     uint32_t row0, int32_t* z, int32_t* err) {
    __shared__ uint32_t sh_w[4];
    __shared__ int sh_i[4];
    __shared__ uint32_t sh_wx;
    const int row = blockIdx.x, tid = threadIdx.x;
    const uint32_t grow = row0 + (uint32_t)row;
    int xr = x[row];
    if (xr < 0 || xr >= V) {
        if (tid == 0 && err) atomicOr(err, DD_DEVERR_TOKEN);
        xr = xr < 0 ? 0 : V - 1;
    }
    uint32_t bw = 0;
    int bi = 0x7FFFFFFF;
    const int nblk = (V + 3) >> 2;
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    for (int b = tid; b < nblk; b += 256) {
        const Words4 W = philox4x32_10((uint32_t)b, grow, step, STREAM_LATENT, k0, k1);
        // branch-free running argmax over v != x (selects; a thread's classes rise with b and e, so
        // an equal word never displaces an earlier class); the word of class x is set aside
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int v = 4 * b + e;
            const uint32_t w = W.w[e];
            const bool take = v < V && v != xr && (w > bw || (w == bw && v < bi));
            bw = take ? w : bw;
            bi = take ? v : bi;
        }
        if ((xr >> 2) == b) sh_wx = W.w[xr & 3];
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const uint32_t w2 = __shfl_xor(bw, o, 64);
        const int i2 = __shfl_xor(bi, o, 64);
        if (w2 > bw || (w2 == bw && i2 < bi)) { bw = w2; bi = i2; }
    }
    if ((tid & 63) == 0) { sh_w[tid >> 6] = bw; sh_i[tid >> 6] = bi; }
    __syncthreads();
    if (tid == 0) {
        for (int k = 1; k < 4; ++k)
            if (sh_w[k] > bw || (sh_w[k] == bw && sh_i[k] < bi)) { bw = sh_w[k]; bi = sh_i[k]; }
        int out = xr;
        if (V > 1) {
            const double sx = at + sigma * word_normal(sh_wx);
            const double sb = sigma * word_normal(bw);
            out = (sx > sb) ? xr : (sx < sb) ? bi : (xr < bi ? xr : bi);
        }
        z[row] = out;
    }
}

dd_status launch_latent(const int32_t* x, int32_t rows, int32_t V, double at, double sigma,
                        uint64_t seed, uint32_t step, uint32_t row0, int32_t* z, int32_t* err,
                        hipStream_t s) {
    if (rows == 0) return DD_OK;
    ProfScope ps(KC_LATENT, s);
    launch_k(latent_kernel, dim3(rows), dim3(256), 0, s, x, V, at, sigma, seed, step, row0,
                       z, err);
    return launch_status("gaussian_latent_argmax");
}

// Element e of tensor `id`: Box-Muller normal from Philox block (e >> 1, id, STREAM_PARAM) words
// 0 and 1 (cosine for even e, sine for odd e); value scale * z + shift in float64, rounded once.
__global__ __launch_bounds__(256) void init_kernel(void* dst, int64_t count, uint32_t id,
                                                   double shift, int is_bf16, uint64_t seed) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= count) return;
    const uint64_t pair = (uint64_t)e >> 1;
    const Words4 W = philox4x32_10((uint32_t)pair, (uint32_t)(pair >> 32), id, STREAM_PARAM,
                                   (uint32_t)seed, (uint32_t)(seed >> 32));
    const double u1 = ((double)W.w[0] + 0.5) * 0x1p-32;
    const double u2 = ((double)W.w[1] + 0.5) * 0x1p-32;
    const double r = sqrt(-2.0 * log(u1));
    const double ang = 2.0 * M_PI * u2;
    const double zz = (e & 1) ? r * sin(ang) : r * cos(ang);
    const double v = 0.02 * zz + shift;
    if (is_bf16) ((bf16_t*)dst)[e] = f64_to_bf16(v);
    else ((float*)dst)[e] = (float)v;
}

dd_status launch_init(void* dst, int64_t count, uint32_t id, double shift, int is_bf16,
                      uint64_t seed, hipStream_t s) {
    if (count == 0) return DD_OK;
    ProfScope ps(KC_INIT, s);
    launch_k(init_kernel, dim3((unsigned)ceil_div(count, 256)), dim3(256), 0, s, dst,
                       count, id, shift, is_bf16, seed);
    return launch_status("init_params");
}

}  // namespace dd
