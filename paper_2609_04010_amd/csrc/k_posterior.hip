// Fused logits -> softmax -> reverse posterior -> two-level Gumbel-max draw.
//
// One workgroup (256 threads) per row.  The row is streamed once from HBM in
// 16-byte chunks; each thread keeps TILE_IT chunks of a tile in registers, so
// the per-wave maximum and the per-group sums of exp(l - max) come from
// registers without a second read.  Only the per-group log-sum-exp values
// (one float per DD_GUMBEL_GROUP classes) go to LDS.  One wavefront then
// finishes the row in fp32: the level-1 draw over the groups, and the level-2
// draw over the 256 logits of the winning group (re-read, an L2 hit).  The
// optional full posterior row (a debug output) comes from a separate kernel in
// float64.
//
// When the vocabulary projection has already produced the per-group
// log-sum-exps (its epilogue computes them from the rounded logits it stores),
// the pass over the row is skipped: one wavefront per row reads the group values
// and the 256 logits of the chosen group only.
//
// The transition is the Psi sampler step (App. A.4, eq. psi-sampler) with correction strength
// kappa; kappa = 1 is the ancestral posterior.  The host folds kappa into the coefficients.
// Masked prior (App. A.1, eq. mdm-posterior; App. A.4, eq. psi-mdm), x = softmax(logits):
//   z_t == mask:  p_v = w_x x_v (v < V), p_mask = w_m; at kappa = 1
//                 w_x = (a_s - a_t)/(1 - a_t), w_m = (1 - a_s)/(1 - a_t)
//   z_t != mask:  kappa = 1: carry-over, z_s = z_t; kappa < 1: keep z_t or remask (probabilities
//                 a_s + kappa (1 - a_s) and the rest).  The row's logits are never read.
// Uniform prior (App. A.2, eq. uniform_true_reverse_posterior; App. A.4, eq. psi-usdm), K = V,
// r = z_t, D = K a_t x_r + 1 - a_t:
//   p_j = [c_x x_j + c_u + u1 D + [j == r](Ka_r x_r + c_z)] / D; at kappa = 1
//   c_x = a_s - a_t, c_z = a_{t|s} - a_t, c_u = (1 - a_{t|s})(1 - a_s)/K, u1 = 0, Ka_r = K a_t.
#include <math.h>

#include "elem.h"
#include "kernels.h"
#include "rng.h"

namespace dd {

constexpr int PT = 256;       // threads per workgroup
#ifndef DD_POST_TILE_IT
#define DD_POST_TILE_IT 4
#endif
constexpr int TILE_IT = DD_POST_TILE_IT;   // 16-byte chunks per thread held in registers per tile
static_assert(TILE_IT >= 1 && TILE_IT <= 32 && (TILE_IT & (TILE_IT - 1)) == 0,
              "the group butterfly needs a power of two no larger than the lanes of a group");

// Wavefront maximum with DPP lane moves (VALU latency) instead of LDS-routed shuffles: two
// quad permutations, the half-row and row mirrors (each row of 16 lanes then holds its maximum),
// then the row broadcasts of lanes 15 and 31; lane 63 ends with the result.
template <int CTRL, int ROW_MASK>
DD_DEV float dpp_max(float v) {
    const int m = __builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), CTRL, ROW_MASK, 0xF, false);
    return fmaxf(v, __int_as_float(m));
}
DD_DEV float wave_max_dpp(float v) {
    v = dpp_max<0xB1, 0xF>(v);    // quad_perm [1, 0, 3, 2]
    v = dpp_max<0x4E, 0xF>(v);    // quad_perm [2, 3, 0, 1]
    v = dpp_max<0x141, 0xF>(v);   // row_half_mirror
    v = dpp_max<0x140, 0xF>(v);   // row_mirror
    v = dpp_max<0x142, 0xA>(v);   // row_bcast15 into rows 1 and 3
    v = dpp_max<0x143, 0xC>(v);   // row_bcast31 into rows 2 and 3
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

// Wavefront argmax of (score, index); the lowest index wins ties; every lane gets the index.
// (Values in and out, with selects: by-reference updates inside branches ended up in scratch.)
DD_DEV int wave_argmax(float s, int i) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float s2 = __shfl_xor(s, o, 64);
        const int i2 = __shfl_xor(i, o, 64);
        const bool take = s2 > s || (s2 == s && i2 < i);
        s = take ? s2 : s;
        i = take ? i2 : i;
    }
    return i;
}

// Stage 0 of the masked prior's draw: the uniform u(w) = (w + 1/2) 2^-32 of the mask group's
// level-1 word (index ngroups of the row's level-1 words), exact in double.  The mask class is
// taken iff u < its probability, which does not depend on the logits (App. A.1: the mask weight
// (1 - a_s)/(1 - a_t), or the Psi form, App. A.4), so the decision can be made before them.
DD_DEV double mask_word_uniform(const uint32_t* noise, int nu, int V, uint64_t seed, uint32_t step,
                                uint32_t grow, int row) {
    const int ngroups = (V + DD_GUMBEL_GROUP - 1) / DD_GUMBEL_GROUP;
    const uint32_t w = noise ? noise[(int64_t)row * nu + ngroups]
                             : counter_word(seed, STREAM_TOP, step, grow, (uint32_t)ngroups);
    return ((double)w + 0.5) * 0x1p-32;
}

// Keep-or-remask draw of an unmasked row (masked prior, kappa < 1): its distribution has only the
// token and the mask, so stage 0 decides.
DD_DEV int32_t keep_or_remask(const PostArgs& a, int row, int zt) {
    return mask_word_uniform(a.noise, a.nu, a.V, a.seed, a.step, a.row0 + (uint32_t)row, row) < a.rmask
               ? a.V : zt;
}

// Level-1 and level-2 draws of one masked (or uniform-prior) row, by one wavefront, from the row's
// per-group log-sum-exps glse[0 .. ngroups) (LDS or global memory) and its logits rowp (read only
// at the chosen group and, uniform prior, at the current token zt).  Row log-sum-exp over the group
// values, level 1 over the groups (4 per lane: one Philox block gives their 4 words) and level 2
// over the 256 classes of the chosen group (4 per lane), all in fp32 with wavefront shuffles.
// With cand (masked prior; the store-free draw) level 2 is the chosen group's candidate, computed
// by the vocabulary projection's epilogue, and the logits are not read.
template <typename T>
DD_DEV void draw_row(const PostArgs& a, int row, int zt, const char* rowp, const float* glse, int lane,
                     const int32_t* cand = nullptr) {
    const int V = a.V;
    const bool mask_prior = a.prior == DD_PRIOR_MASK;
    const int ngroups = (V + DD_GUMBEL_GROUP - 1) / DD_GUMBEL_GROUP;
    const uint32_t grow = a.row0 + (uint32_t)row;
    float m = -INFINITY;
    for (int g = lane; g < ngroups; g += 64) m = fmaxf(m, glse[g]);
    m = wave_max(m);
    const float mref = isinf(m) ? 0.f : m;
    float sum = 0.f;
    for (int g = lane; g < ngroups; g += 64) sum += expf(glse[g] - mref);
    const float lse = mref + logf(wave_sum(sum));

    float c_r = 0.f, Dn = 1.f, c_u = 0.f;
    if (!mask_prior) {   // uniform prior: x_r enters the mass of the current token's class
        const float xr = expf(Elem<T>::load1(rowp, zt) - lse);
        c_r = (float)a.Ka_r * xr + (float)a.c_z;
        Dn = (float)a.Ka_t * xr + (float)a.one_m_at;
        c_u = (float)a.c_u + (float)a.u1 * Dn;
    }
    const float log_wx = (float)a.log_wx;
    const float c_x = (float)a.c_x, log_dn = logf(Dn);
    const uint32_t k0 = (uint32_t)a.seed, k1 = (uint32_t)(a.seed >> 32);

    // stage 0 (mask prior): the mask class is taken iff the mask word's uniform is below w_m (a row
    // without a finite log-sum-exp goes on to be reported below)
    if (mask_prior && isfinite(lse) && mask_word_uniform(a.noise, a.nu, V, a.seed, a.step, grow, row) < a.wm) {
        if (lane == 0) {
            a.z_s[row] = V;
            if (a.row_lse) a.row_lse[row] = lse;
        }
        return;
    }

    // level 1 over the real groups: group g has log mass log w_x + lse_g - lse (mask prior) or
    // log((c_x X_g + n_g c_u + [r in g] c_r) / D) (uniform prior)
    float best = -INFINITY;
    int bi = 0x7FFFFFFF;
    for (int gb = 0; gb < ngroups; gb += 256) {
        const int base = gb + 4 * lane;
        if (base >= ngroups) break;
        uint32_t wd[4];
        if (a.noise) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                wd[i] = (base + i < ngroups) ? a.noise[(int64_t)row * a.nu + base + i] : 0u;
        } else {
            const Words4 W = philox4x32_10((uint32_t)(base >> 2), grow, a.step, STREAM_TOP, k0, k1);
#pragma unroll
            for (int i = 0; i < 4; ++i) wd[i] = W.w[i];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int g = base + i;
            if (g >= ngroups) continue;
            float logm;
            if (mask_prior) {
                logm = log_wx + (glse[g] - lse);
            } else {
                const int lo = g * DD_GUMBEL_GROUP;
                const int n = min(DD_GUMBEL_GROUP, V - lo);
                const float X = expf(glse[g] - lse);
                logm = logf(c_x * X + (float)n * c_u + ((zt >= lo && zt < lo + n) ? c_r : 0.f)) - log_dn;
            }
            const float sc = logm + word_gumbel_f(wd[i]);
            const bool take = sc > best || (sc == best && g < bi);
            best = take ? sc : best;
            bi = take ? g : bi;
        }
    }
    const int gstar = wave_argmax(best, bi);

    int result = V;
    if (gstar >= ngroups || !isfinite(lse)) {
        // no group had a valid score (NaN or +inf logits, or no finite logit): the row keeps
        // its token and the caller is told; gstar must not index anything
        result = -1;
    } else if (cand) {   // level 2 by the group's candidate
        const int c = cand[gstar], lo = gstar * DD_GUMBEL_GROUP;
        result = (c >= lo && c < min(V, lo + DD_GUMBEL_GROUP)) ? c : -1;
    } else {   // level 2 inside the chosen group
        best = -INFINITY;
        bi = 0x7FFFFFFF;
        const int base = gstar * DD_GUMBEL_GROUP + 4 * lane;
        if (base < V) {
            uint32_t wd[4];
            if (a.noise) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    wd[i] = (base + i < V) ? a.noise[(int64_t)row * a.nu + a.ntop + base + i] : 0u;
            } else {
                const Words4 W = philox4x32_10((uint32_t)(base >> 2), grow, a.step, STREAM_CLASS, k0, k1);
#pragma unroll
                for (int i = 0; i < 4; ++i) wd[i] = W.w[i];
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int j = base + i;
                if (j >= V) continue;
                const float l = Elem<T>::load1(rowp, j);
                float logp;
                if (mask_prior) logp = log_wx + (l - lse);
                else logp = logf(c_x * expf(l - lse) + c_u + (j == zt ? c_r : 0.f)) - log_dn;
                const float sc = logp + word_gumbel_f(wd[i]);
                const bool take = sc > best || (sc == best && j < bi);
                best = take ? sc : best;
                bi = take ? j : bi;
            }
        }
        result = wave_argmax(best, bi);
        if (result >= V) result = -1;           // no class of the group had a valid score
    }
    if (result < 0) {
        if (lane == 0 && a.err) atomicOr(a.err, DD_DEVERR_LOGITS);
        result = zt;
    }
    if (lane == 0) {
        a.z_s[row] = result;
        if (a.row_lse) a.row_lse[row] = lse;
    }
}

// The row's current token into zt (an id outside the K classes is flagged and clamped).  Returns
// false when the row is settled without its logits: masked prior, unmasked row (carry-over, or
// keep/remask under kappa < 1), whose z_s the leader thread has written.
DD_DEV bool row_needs_draw(const PostArgs& a, int row, bool leader, int& zt) {
    const int V = a.V;
    const bool mask_prior = a.prior == DD_PRIOR_MASK;
    const int K = mask_prior ? V + 1 : V;
    zt = a.z_t[row];
    if (zt < 0 || zt >= K) {
        if (leader && a.err) atomicOr(a.err, DD_DEVERR_TOKEN);
        zt = zt < 0 ? 0 : K - 1;
    }
    if (mask_prior && zt != V) {
        if (leader) a.z_s[row] = a.remask ? keep_or_remask(a, row, zt) : zt;
        return false;
    }
    return true;
}

template <typename T>
__global__ __launch_bounds__(PT) void posterior_kernel(PostArgs a) {
    extern __shared__ float s_lse[];  // one log-sum-exp per group

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
    int zt;
    if (!row_needs_draw(a, row, tid == 0, zt)) return;

    const char* rowp = (const char*)a.logits + (size_t)blockIdx.x * (size_t)a.ld * sizeof(T);
    const int nchunk = (V + E - 1) / E;

    // ---- pass over the row: per-group log-sum-exp ---------------------------------------
    // Elements past V count as -inf: chunks past the row are filled with -inf bits, and the one
    // ragged chunk (V not a multiple of E) is clipped in registers.  Each lane ends a tile with TILE_IT
    // partial sums (one per iteration, i.e. per group slice); a butterfly over the LPG lanes of a
    // group halves the list at every step, so TILE_IT sums cost log2(LPG) steps and TILE_IT
    // shuffles in total instead of TILE_IT * log2(LPG).
    // tiles of TILE_IT * PT chunks; the loads of the next tile are issued before the current one
    // is reduced (two register buffers), so a wavefront always has a tile in flight
    auto load_tile = [&](uint4 (&buf)[TILE_IT], const int tile0) {
        if ((tile0 + TILE_IT * PT) * E <= V) {   // every element of the tile is in the row
#pragma unroll
            for (int it = 0; it < TILE_IT; ++it)
                buf[it] = *(const uint4*)(rowp + (size_t)(tile0 + it * PT + tid) * 16);
        } else {   // last tile: clamped loads, -inf past the row, the ragged chunk clipped
#pragma unroll
            for (int it = 0; it < TILE_IT; ++it) {
                const int c = tile0 + it * PT + tid;
                const uint4 x = *(const uint4*)(rowp + (size_t)min(c, nchunk - 1) * 16);
                buf[it] = (c < nchunk) ? x : Elem<T>::NEG_INF4;
            }
            if (V % E != 0) {
#pragma unroll
                for (int it = 0; it < TILE_IT; ++it)
                    if (tile0 + it * PT + tid == nchunk - 1) Elem<T>::clip(buf[it], V % E);
            }
        }
    };
    auto reduce_tile = [&](uint4 (&buf)[TILE_IT], const int tile0) {
        float m = -INFINITY;
#pragma unroll
        for (int it = 0; it < TILE_IT; ++it)
#pragma unroll
            for (int e = 0; e < E; ++e) m = fmaxf(m, Elem<T>::get(buf[it], e));
        m = wave_max_dpp(m);
        const float mref = (m == -INFINITY) ? 0.f : m;
        const float moff = -mref * LOG2E;
        float v[TILE_IT];
#pragma unroll
        for (int it = 0; it < TILE_IT; ++it) {
            float sum = 0.f;
#pragma unroll
            for (int e = 0; e < E; ++e) sum += __builtin_amdgcn_exp2f(fmaf(Elem<T>::get(buf[it], e), LOG2E, moff));
            v[it] = sum;
        }
        int idx = 0;   // iteration whose group sum this lane holds at the end
#pragma unroll
        for (int o = LPG / 2, n = TILE_IT; o >= 1; o >>= 1) {
            if (n > 1) {
                n >>= 1;
                const bool up = (lane & o) != 0;
                // the swap is written with bit masks: as a select of two array elements the compiler
                // turns it into a dynamically indexed register array (a compare-select chain)
                const uint32_t mk = up ? 0xFFFFFFFFu : 0u;
#pragma unroll
                for (int i = 0; i < TILE_IT / 2; ++i) {
                    if (i < n) {
                        const uint32_t lo = __float_as_uint(v[i]), hi = __float_as_uint(v[n + i]);
                        const float send = __uint_as_float((lo & mk) | (hi & ~mk));
                        const float keep = __uint_as_float((hi & mk) | (lo & ~mk));
                        v[i] = keep + __shfl_xor(send, o, 64);
                    }
                }
                if (up) idx += n;
            } else {
                v[0] += __shfl_xor(v[0], o, 64);
            }
        }
        constexpr int DUP = (LPG / TILE_IT) > 1 ? LPG / TILE_IT : 1;   // lanes holding the same sum
        if ((lane & (DUP - 1)) == 0) {
            const int c = tile0 + idx * PT + (tid & ~(LPG - 1));
            if (c < nchunk) s_lse[c / LPG] = mref + logf(v[0]);
        }
    };
    constexpr int TS = TILE_IT * PT;
    uint4 ba[TILE_IT], bb[TILE_IT];
    load_tile(ba, 0);
    for (int t0 = 0; t0 < nchunk; t0 += 2 * TS) {
        const bool next_b = t0 + TS < nchunk;
        if (next_b) load_tile(bb, t0 + TS);
        reduce_tile(ba, t0);
        if (!next_b) break;
        if (t0 + 2 * TS < nchunk) load_tile(ba, t0 + 2 * TS);
        reduce_tile(bb, t0 + TS);
    }
    __syncthreads();

    // ---- tail: one wavefront finishes the row (no further workgroup barrier); the other
    // wavefronts leave
    if ((tid >> 6) != 0) return;
    draw_row<T>(a, row, zt, rowp, s_lse, lane);
}

// Rows whose per-group log-sum-exps came with the logits (the vocabulary projection's group
// log-sum-exp epilogue): one wavefront per row, four rows per workgroup, and no pass over the row.
template <typename T>
__global__ __launch_bounds__(256) void posterior_grouped_kernel(PostArgs a) {
    const int lane = threadIdx.x & 63;
    const int j = (int)blockIdx.x * 4 + (int)(threadIdx.x >> 6);   // logits row
    int row = j;
    if (a.count) {
        if (j >= *a.count) return;
        row = a.rows_idx[j];
    } else if (j >= a.rows) {
        return;
    }
    int zt;
    if (!row_needs_draw(a, row, lane == 0, zt)) return;
    const char* rowp = a.logits ? (const char*)a.logits + (size_t)j * (size_t)a.ld * sizeof(T) : nullptr;
    draw_row<T>(a, row, zt, rowp, a.glse + (int64_t)j * a.glse_ld, lane,
                a.cand ? a.cand + (int64_t)j * a.cand_ld : nullptr);
}

// Debug output: the full posterior row in float64 arithmetic (two passes over the logits).
template <typename T>
__global__ __launch_bounds__(PT) void posterior_probs_kernel(PostArgs a) {
    __shared__ double sh[PT / 64];
    const int row = blockIdx.x, tid = threadIdx.x;
    const int V = a.V;
    const bool mask_prior = a.prior == DD_PRIOR_MASK;
    const int K = mask_prior ? V + 1 : V;
    int zt = a.z_t[row];
    zt = zt < 0 ? 0 : (zt >= K ? K - 1 : zt);
    float* out = a.probs + (int64_t)row * K;
    if (mask_prior && zt != V) {
        const double keep = a.remask ? a.keep : 1.0, rm = a.remask ? a.rmask : 0.0;
        for (int j = tid; j < K; j += PT) out[j] = (j == zt) ? (float)keep : (j == V ? (float)rm : 0.f);
        return;
    }
    const char* rowp = (const char*)a.logits + (size_t)row * (size_t)a.ld * sizeof(T);
    double m = -INFINITY;
    for (int j = tid; j < V; j += PT) m = fmax(m, (double)Elem<T>::load1(rowp, j));
    for (int o = 32; o > 0; o >>= 1) m = fmax(m, __shfl_xor(m, o, 64));
    if ((tid & 63) == 0) sh[tid >> 6] = m;
    __syncthreads();
    m = fmax(fmax(sh[0], sh[1]), fmax(sh[2], sh[3]));
    __syncthreads();
    double sum = 0.0;
    for (int j = tid; j < V; j += PT) sum += exp((double)Elem<T>::load1(rowp, j) - m);
    for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o, 64);
    if ((tid & 63) == 0) sh[tid >> 6] = sum;
    __syncthreads();
    const double lse = m + log(sh[0] + sh[1] + sh[2] + sh[3]);
    double c_r = 0.0, Dn = 1.0, c_u = 0.0;
    if (!mask_prior) {
        const double xr = exp((double)Elem<T>::load1(rowp, zt) - lse);
        c_r = a.Ka_r * xr + a.c_z;
        Dn = a.Ka_t * xr + a.one_m_at;
        c_u = a.c_u + a.u1 * Dn;
    }
    for (int j = tid; j < K; j += PT) {
        double p;
        if (mask_prior) {
            p = (j < V) ? a.wx * exp((double)Elem<T>::load1(rowp, j) - lse) : a.wm;
        } else {
            const double x = exp((double)Elem<T>::load1(rowp, j) - lse);
            p = (a.c_x * x + c_u + (j == zt ? c_r : 0.0)) / Dn;
        }
        out[j] = (float)p;
    }
}

// Keep-or-remask draws of all unmasked rows (masked prior, kappa < 1), one thread per row; masked
// rows are left untouched (the posterior kernel draws them).
__global__ __launch_bounds__(256) void remask_kernel(PostArgs a) {
    const int row = blockIdx.x * 256 + threadIdx.x;
    if (row >= a.rows) return;
    int zt = a.z_t[row];
    if (zt == a.V) return;
    if (zt < 0 || zt > a.V) {   // flagged; ids past the mask count as masked (left to the posterior)
        if (a.err) atomicOr(a.err, DD_DEVERR_TOKEN);
        if (zt > a.V) return;
        zt = 0;
    }
    a.z_s[row] = keep_or_remask(a, row, zt);
}

dd_status launch_remask(const PostArgs& a, hipStream_t s) {
    if (a.rows == 0) return DD_OK;
    ProfScope ps(KC_POSTERIOR, s);
    launch_k(remask_kernel, dim3((a.rows + 255) / 256), dim3(256), 0, s, a);
    return launch_status("remask");
}

// Ascending list of the rows whose token is the mask id, and its length.  One workgroup walks the
// tokens in blocks of 4 per thread (16-byte loads when z is 16-byte aligned): each thread counts its 4
// flags, an inclusive shuffle scan gives the offsets inside the wavefront, the 16 wavefront totals go
// through LDS, and every thread writes its rows after the rows of earlier threads and blocks.
constexpr int CT = 1024;

// stage 0 of the masked prior's draw taken ahead of the logits (see mask_word_uniform)
struct PreDraw {
    const uint32_t* noise;
    int nu, V, on;
    uint64_t seed;
    uint32_t step, row0;
    double wm;
};

__global__ __launch_bounds__(CT) void compact_masked_kernel(const int32_t* z, int64_t M,
                                                            int32_t mask_id, int32_t* idx,
                                                            int32_t* count, int L, int32_t* seq,
                                                            PreDraw pd) {
    __shared__ int wsum[CT / 64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const bool vec = ((uintptr_t)z & 15) == 0;
    int base = 0;   // rows listed by earlier blocks (the same in every thread)
    const float inv_l = seq ? 1.0f / (float)L : 0.f;
    for (int64_t b0 = 0; b0 < M; b0 += 4 * CT) {
        const int64_t i0 = b0 + 4 * (int64_t)tid;
        // the first sequence start at or after row i0: row nb of sequence sq (a float quotient, at
        // most two below ceil(i0 / L), then raised to it; independent of the load below)
        int64_t nb = 0;
        int sq = 0;
        if (seq) {
            sq = max((int)((float)i0 * inv_l) - 1, 0);
#pragma unroll
            for (int k = 0; k < 3; ++k) sq += (int64_t)sq * L < i0;
            nb = (int64_t)sq * L;
        }
        int f[4];
        if (vec && i0 + 3 < M) {
            const int4 v = *(const int4*)(z + i0);
            f[0] = v.x == mask_id; f[1] = v.y == mask_id; f[2] = v.z == mask_id; f[3] = v.w == mask_id;
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) f[e] = (i0 + e < M) && z[i0 + e] == mask_id;
        }
        if (pd.on) {
            // a masked row that stage 0 keeps masked needs no logits: it is not listed
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (f[e]) {
                    const int r = (int)i0 + e;
                    f[e] = !(mask_word_uniform(pd.noise, pd.nu, pd.V, pd.seed, pd.step, pd.row0 + (uint32_t)r, r) <
                             pd.wm);
                }
        }
        const int c = f[0] + f[1] + f[2] + f[3];
        int incl = c;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int t = __shfl_up(incl, o, 64);
            if (lane >= o) incl += t;
        }
        if (lane == 63) wsum[wave] = incl;
        __syncthreads();
        int before = 0, total = 0;
#pragma unroll
        for (int w = 0; w < CT / 64; ++w) {
            const int v = wsum[w];
            before += w < wave ? v : 0;
            total += v;
        }
        int pos = base + before + incl - c;
        if (seq) {
            // a sequence that starts at one of this thread's rows starts at list index pos + (rows
            // listed before it among the four)
            int p = pos;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if (i0 + e == nb && nb < M) {
                    seq[sq++] = p;
                    nb += L;
                }
                p += f[e];
            }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (f[e]) idx[pos++] = (int32_t)(i0 + e);
        base += total;
        __syncthreads();   // wsum is rewritten by the next block
    }
    if (tid == 0) {
        *count = base;
        if (seq) seq[M / L] = base;
    }
}

dd_status launch_compact(const int32_t* z, int64_t M, int32_t mask_id, int32_t* idx, int32_t* count,
                         hipStream_t s, int L, int32_t* seq, const PostArgs* pre) {
    if (seq && (L <= 0 || M % L != 0)) {
        set_error("sequence starts need rows of L > 0 tokens (M = %lld, L = %d)", (long long)M, L);
        return DD_E_ARG;
    }
    ProfScope ps(KC_COMPACT, s);
    PreDraw pd = {};
    if (pre) {
        if (pre->prior != DD_PRIOR_MASK || mask_id != pre->V) {
            set_error("the stage-0 pre-draw needs the masked prior with the mask id V");
            return DD_E_ARG;
        }
        pd = {pre->noise, pre->nu, pre->V, 1, pre->seed, pre->step, pre->row0, pre->wm};
    }
    launch_k(compact_masked_kernel, dim3(1), dim3(CT), 0, s, z, M, mask_id, idx, count, L, seq, pd);
    return launch_status("compact_masked");
}

dd_status launch_posterior(const PostArgs& a, int logits_dtype, hipStream_t s) {
    if (a.rows == 0) return DD_OK;
    const int ngroups = (a.V + DD_GUMBEL_GROUP - 1) / DD_GUMBEL_GROUP;
    const size_t shmem = (size_t)ngroups * sizeof(float);
    {
        ProfScope ps(KC_POSTERIOR, s);
        const dim3 g4((unsigned)((a.rows + 3) / 4));
        if (a.glse && logits_dtype == DD_BF16)
            launch_k(posterior_grouped_kernel<bf16_t>, g4, dim3(256), 0, s, a);
        else if (a.glse)
            launch_k(posterior_grouped_kernel<float>, g4, dim3(256), 0, s, a);
        else if (logits_dtype == DD_BF16)
            launch_k(posterior_kernel<bf16_t>, dim3(a.rows), dim3(PT), shmem, s, a);
        else
            launch_k(posterior_kernel<float>, dim3(a.rows), dim3(PT), shmem, s, a);
    }
    if (a.probs && !a.count) {
        if (logits_dtype == DD_BF16)
            launch_k(posterior_probs_kernel<bf16_t>, dim3(a.rows), dim3(PT), 0, s, a);
        else
            launch_k(posterior_probs_kernel<float>, dim3(a.rows), dim3(PT), 0, s, a);
    }
    return launch_status("posterior");
}

}  // namespace dd
