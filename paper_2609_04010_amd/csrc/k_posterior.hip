// Fused logits -> softmax -> reverse posterior -> two-level Gumbel-max draw.
//
// One workgroup (256 threads) per row.  The row is streamed once from HBM in
// 16-byte chunks; each thread keeps up to 16 chunks of a tile in registers, so
// the per-wave maximum and the per-group sums of exp(l - max) come from
// registers without a second read.  Only the per-group log-sum-exp values
// (one float per DD_GUMBEL_GROUP classes) go to LDS.  The level-1 draw then
// runs over the groups, and the level-2 draw re-reads the 256 logits of the
// winning group (an L2 hit).
//
// Masked prior (App. A.1, eq. mdm-posterior, x = softmax(logits)):
//   z_t == mask:  p_v = w_x x_v (v < V), p_mask = w_m,
//                 w_x = (a_s - a_t)/(1 - a_t), w_m = (1 - a_s)/(1 - a_t)
//   z_t != mask:  carry-over, z_s = z_t (the row is not read).
// Uniform prior (App. A.2, eq. uniform_true_reverse_posterior), K = V, r = z_t:
//   p_j = [c_x x_j + c_u + [j == r](K a_t x_r + c_z)] / (K a_t x_r + 1 - a_t)
//   c_x = a_s - a_t, c_z = a_{t|s} - a_t, c_u = (1 - a_{t|s})(1 - a_s)/K.
#include <math.h>

#include "kernels.h"
#include "rng.h"

namespace dd {

constexpr int PT = 256;       // threads per workgroup
constexpr int TILE_IT = 16;   // 16-byte chunks per thread held in registers per tile
constexpr float LOG2E = 1.4426950408889634f;

template <typename T> struct Elem;
template <> struct Elem<bf16_t> {
    static constexpr int E = 8;  // elements per 16-byte chunk
    DD_DEV static float get(const uint4& c, int e) {
        const uint32_t w = (e < 2) ? c.x : (e < 4) ? c.y : (e < 6) ? c.z : c.w;
        return (e & 1) ? bf16_hi(w) : bf16_lo(w);
    }
    DD_DEV static float load1(const void* p, int64_t i) { return bf16_to_f32(((const bf16_t*)p)[i]); }
};
template <> struct Elem<float> {
    static constexpr int E = 4;
    DD_DEV static float get(const uint4& c, int e) {
        const uint32_t w = (e == 0) ? c.x : (e == 1) ? c.y : (e == 2) ? c.z : c.w;
        return __uint_as_float(w);
    }
    DD_DEV static float load1(const void* p, int64_t i) { return ((const float*)p)[i]; }
};

DD_DEV void better(double& s, int& i, double s2, int i2) {
    if (s2 > s || (s2 == s && i2 < i)) { s = s2; i = i2; }
}

// Block-wide argmax of (score, index); the lowest index wins ties.  Result in lane 0 of every wave
// is broadcast through LDS to all threads.
DD_DEV void block_argmax(double& s, int& i, double* sh_s, int* sh_i) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        double s2 = __shfl_xor(s, o, 64);
        int i2 = __shfl_xor(i, o, 64);
        better(s, i, s2, i2);
    }
    const int w = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) { sh_s[w] = s; sh_i[w] = i; }
    __syncthreads();
    s = sh_s[0]; i = sh_i[0];
#pragma unroll
    for (int k = 1; k < PT / 64; ++k) better(s, i, sh_s[k], sh_i[k]);
}

DD_DEV double block_max_d(double v, double* sh) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, 64));
    __syncthreads();
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
    __syncthreads();
    double r = sh[0];
#pragma unroll
    for (int k = 1; k < PT / 64; ++k) r = fmax(r, sh[k]);
    return r;
}

DD_DEV double block_sum_d(double v, double* sh) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
    __syncthreads();
    double r = sh[0];
#pragma unroll
    for (int k = 1; k < PT / 64; ++k) r += sh[k];
    return r;
}

template <typename T>
__global__ __launch_bounds__(PT) void posterior_kernel(PostArgs a) {
    extern __shared__ float s_lse[];  // one log-sum-exp per group
    __shared__ double sh_d[PT / 64];
    __shared__ int sh_i[PT / 64];

    constexpr int E = Elem<T>::E;
    constexpr int LPG = DD_GUMBEL_GROUP / E;  // lanes per group (32 bf16, 64 fp32)
    int row = blockIdx.x;                     // token row; the logits row is blockIdx.x
    if (a.count) {                            // compacted: logits row j holds token row rows_idx[j]
        if ((int)blockIdx.x >= *a.count) return;
        row = a.rows_idx[blockIdx.x];
    }
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int V = a.V;
    const bool mask_prior = a.prior == DD_PRIOR_MASK;
    const int K = mask_prior ? V + 1 : V;
    const uint32_t grow = a.row0 + (uint32_t)row;

    int zt = a.z_t[row];
    if (zt < 0 || zt >= K) {
        if (tid == 0 && a.err) atomicOr(a.err, DD_DEVERR_TOKEN);
        zt = zt < 0 ? 0 : K - 1;
    }
    if (mask_prior && zt != V) {  // carry-over: the row's logits are never read
        if (tid == 0) a.z_s[row] = zt;
        if (a.probs)
            for (int j = tid; j < K; j += PT) a.probs[(int64_t)row * K + j] = (j == zt) ? 1.f : 0.f;
        return;
    }

    const char* rowp = (const char*)a.logits + (size_t)blockIdx.x * (size_t)a.ld * sizeof(T);
    const int nchunk = (V + E - 1) / E;
    const int ngroups = (V + DD_GUMBEL_GROUP - 1) / DD_GUMBEL_GROUP;

    // ---- pass over the row: per-group log-sum-exp ---------------------------------------
    for (int tile0 = 0; tile0 < nchunk; tile0 += TILE_IT * PT) {
        uint4 buf[TILE_IT];
#pragma unroll
        for (int it = 0; it < TILE_IT; ++it) {
            const int c = tile0 + it * PT + tid;
            if (c < nchunk) buf[it] = *(const uint4*)(rowp + (size_t)c * 16);
            else buf[it] = make_uint4(0u, 0u, 0u, 0u);
        }
        float m = -INFINITY;
#pragma unroll
        for (int it = 0; it < TILE_IT; ++it) {
            const int c = tile0 + it * PT + tid;
#pragma unroll
            for (int e = 0; e < E; ++e)
                if (c * E + e < V) m = fmaxf(m, Elem<T>::get(buf[it], e));
        }
        m = wave_max(m);
        const float mref = (m == -INFINITY) ? 0.f : m;
        const float moff = -mref * LOG2E;
        float part[TILE_IT];
#pragma unroll
        for (int it = 0; it < TILE_IT; ++it) {
            const int c = tile0 + it * PT + tid;
            float s = 0.f;
#pragma unroll
            for (int e = 0; e < E; ++e)
                if (c * E + e < V) s += __builtin_amdgcn_exp2f(fmaf(Elem<T>::get(buf[it], e), LOG2E, moff));
            part[it] = s;
        }
#pragma unroll
        for (int it = 0; it < TILE_IT; ++it) {
#pragma unroll
            for (int o = LPG / 2; o > 0; o >>= 1) part[it] += __shfl_xor(part[it], o, 64);
        }
        if ((lane % LPG) == 0) {
#pragma unroll
            for (int it = 0; it < TILE_IT; ++it) {
                const int c = tile0 + it * PT + tid;
                if (c < nchunk) s_lse[c / LPG] = mref + logf(part[it]);
            }
        }
    }
    __syncthreads();

    // ---- row log-sum-exp ---------------------------------------------------------------
    double lmax = -INFINITY;
    for (int g = tid; g < ngroups; g += PT) lmax = fmax(lmax, (double)s_lse[g]);
    lmax = block_max_d(lmax, sh_d);
    const double lref = isinf(lmax) ? 0.0 : lmax;
    double lsum = 0.0;
    for (int g = tid; g < ngroups; g += PT) lsum += exp((double)s_lse[g] - lref);
    lsum = block_sum_d(lsum, sh_d);
    const double lse = lref + log(lsum);

    // uniform prior: x_r and the row-specific coefficients
    double c_r = 0.0, Dn = 1.0;
    if (!mask_prior) {
        const double xr = exp((double)Elem<T>::load1(rowp, zt) - lse);
        c_r = a.Ka_t * xr + a.c_z;
        Dn = a.Ka_t * xr + a.one_m_at;
    }

    // ---- level 1: choose a group ------------------------------------------------------
    double best = -INFINITY;
    int bi = 0x7FFFFFFF;
    for (int g = tid; g < a.ntop; g += PT) {
        double logm;
        if (mask_prior) {
            logm = (g < ngroups) ? a.log_wx + ((double)s_lse[g] - lse) : a.log_wm;
        } else {
            const int lo = g * DD_GUMBEL_GROUP;
            const int n = min(DD_GUMBEL_GROUP, V - lo);
            const double X = exp((double)s_lse[g] - lse);
            const double M = a.c_x * X + n * a.c_u + ((zt >= lo && zt < lo + n) ? c_r : 0.0);
            logm = log(M / Dn);
        }
        const uint32_t w = a.noise ? a.noise[(int64_t)row * a.nu + g]
                                   : counter_word(a.seed, STREAM_TOP, a.step, grow, (uint32_t)g);
        better(best, bi, logm + word_gumbel(w), g);
    }
    block_argmax(best, bi, sh_d, sh_i);
    const int gstar = bi;

    // ---- level 2: choose a class inside the group ---------------------------------------
    int result;
    if (mask_prior && gstar == ngroups) {
        result = V;
    } else {
        best = -INFINITY;
        bi = 0x7FFFFFFF;
        const int j = gstar * DD_GUMBEL_GROUP + tid;
        if (j < V) {
            const double l = (double)Elem<T>::load1(rowp, j);
            double logp;
            if (mask_prior) {
                logp = a.log_wx + (l - lse);
            } else {
                const double x = exp(l - lse);
                logp = log((a.c_x * x + a.c_u + (j == zt ? c_r : 0.0)) / Dn);
            }
            const uint32_t w = a.noise ? a.noise[(int64_t)row * a.nu + a.ntop + j]
                                       : counter_word(a.seed, STREAM_CLASS, a.step, grow, (uint32_t)j);
            best = logp + word_gumbel(w);
            bi = j;
        }
        block_argmax(best, bi, sh_d, sh_i);
        result = bi;
    }
    if (tid == 0) a.z_s[row] = result;

    if (a.probs) {  // debug output of the full posterior row
        for (int j = tid; j < K; j += PT) {
            double p;
            if (mask_prior) {
                p = (j < V) ? a.wx * exp((double)Elem<T>::load1(rowp, j) - lse) : a.wm;
            } else {
                const double x = exp((double)Elem<T>::load1(rowp, j) - lse);
                p = (a.c_x * x + a.c_u + (j == zt ? c_r : 0.0)) / Dn;
            }
            a.probs[(int64_t)row * K + j] = (float)p;
        }
    }
}

// Ascending list of the rows whose token is the mask id, and its length (one workgroup: each thread
// counts a contiguous slice, a workgroup scan gives the slice offsets, then the slices are written).
constexpr int CT = 1024;

__global__ __launch_bounds__(CT) void compact_masked_kernel(const int32_t* z, int64_t M,
                                                            int32_t mask_id, int32_t* idx,
                                                            int32_t* count) {
    __shared__ int sh[CT];
    const int tid = threadIdx.x;
    const int64_t per = (M + CT - 1) / CT;
    const int64_t lo = (int64_t)tid * per, hi = lo + per < M ? lo + per : M;
    int c = 0;
    for (int64_t r = lo; r < hi; ++r) c += (z[r] == mask_id);
    sh[tid] = c;
    __syncthreads();
    for (int off = 1; off < CT; off <<= 1) {
        const int v = tid >= off ? sh[tid - off] : 0;
        __syncthreads();
        sh[tid] += v;
        __syncthreads();
    }
    int pos = sh[tid] - c;
    for (int64_t r = lo; r < hi; ++r)
        if (z[r] == mask_id) idx[pos++] = (int32_t)r;
    if (tid == CT - 1) *count = sh[CT - 1];
}

dd_status launch_compact(const int32_t* z, int64_t M, int32_t mask_id, int32_t* idx, int32_t* count,
                         hipStream_t s) {
    ProfScope ps(KC_COMPACT, s);
    hipLaunchKernelGGL(compact_masked_kernel, dim3(1), dim3(CT), 0, s, z, M, mask_id, idx, count);
    return launch_status("compact_masked");
}

dd_status launch_posterior(const PostArgs& a, int logits_dtype, hipStream_t s) {
    if (a.rows == 0) return DD_OK;
    const int ngroups = (a.V + DD_GUMBEL_GROUP - 1) / DD_GUMBEL_GROUP;
    const size_t shmem = (size_t)ngroups * sizeof(float);
    ProfScope ps(KC_POSTERIOR, s);
    if (logits_dtype == DD_BF16)
        hipLaunchKernelGGL(posterior_kernel<bf16_t>, dim3(a.rows), dim3(PT), shmem, s, a);
    else
        hipLaunchKernelGGL(posterior_kernel<float>, dim3(a.rows), dim3(PT), shmem, s, a);
    return launch_status("posterior");
}

}  // namespace dd
