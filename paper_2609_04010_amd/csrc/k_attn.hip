// Multi-head attention softmax(q k^T / sqrt(dh)) v, flash style (no L x L tensor), over every key
// or, with a visibility pattern, over the keys j of query i with j < pre_i or lo_i <= j < hi_i (a
// prefix plus one window: bidirectional, causal, block-causal and the [x, z_1] block-diffusion
// pattern all take this form).
//
// bf16 path (dh = 64): a workgroup of 4 wavefronts owns 128 queries of one (batch, head); each
// wavefront owns 32 queries.  Key/value tiles of 64 tokens are staged in LDS (double-buffered,
// prefetched through registers): K row-major (padded rows), V transposed so the P.V contraction
// reads contiguous 16-byte fragments.
//   S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (first operand: K rows from LDS; second: the wave's
//         Q fragment, held in registers for the whole kernel).  Each lane then holds 32 scores of
//         one query, the other 32 of the tile being in lane ^ 32.
//   Online softmax in base 2 with the 1/sqrt(dh) scale folded into the exponent; the row max is
//         combined with one cross-lane exchange; the running sum stays per lane until the end.
//   O^T += V^T P^T: the probabilities are rounded to bf16 and used directly as the second MFMA
//         operand (no shuffles: the key order of V^T in LDS is permuted to match the accumulator
//         layout of S^T), so each lane's output column is again its own query.
// Patterns (MASKED instance): a workgroup visits only the key tiles that meet the union of its
// queries' visible sets (the prefix tiles, then the window tiles); a wavefront whose queries see
// nothing of a tile skips its arithmetic; a tile that every query of the wavefront sees whole takes
// no per-element test.  Rows that have seen no visible key yet keep mref = -inf and use exponent
// reference 0, so their probabilities are exactly 0 until their first visible key.
// fp32 path (validation): one thread per (batch, head, query), fp32 online softmax.
#include <limits.h>
#include <math.h>

#include <algorithm>

#include "kernels.h"

namespace dd {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;

constexpr int AQ = 128;  // queries per workgroup
constexpr int AK = 64;   // keys per tile
constexpr int DH = 64;
constexpr int KSTR = DH + 8;
constexpr int VSTR = AK + 8;

// Key order inside a transposed V row: within each 16-key step s the MFMA operand slots of lane
// group g hold keys 16s + 4g + {0..3} and 16s + 8 + 4g + {0..3}; those eight keys are stored
// contiguously at positions 16s + 8g .. + 7 (key 16s + 4g + 8h + r at position 16s + 8g + 4h + r),
// so each lane reads its operand with one 16-byte load.

DD_DEV int wave_max_i(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, 64));
    return v;
}
DD_DEV int wave_min_i(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, 64));
    return v;
}

// The visible set of query qi (< L): (pre, lo, hi) read from the pattern, an invalid entry
// reported and replaced by "every key".
DD_DEV void query_window(const AttnArgs& a, int qi, int& pre, int& lo, int& hi) {
    const int L = a.L;
    pre = a.mask[qi];
    lo = a.mask[L + qi];
    hi = a.mask[2 * L + qi];
    const bool ok = pre >= 0 && pre <= L && lo >= 0 && lo <= hi && hi <= L && (pre > 0 || hi > lo);
    if (!ok) {
        if (a.err) atomicOr(a.err, DD_DEVERR_MASK);
        pre = L;
        lo = hi = 0;
    }
}

template <bool MASKED>
__global__ __launch_bounds__(256) void attn_bf16_kernel(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) bf16_t Ks[2][AK * KSTR];
    __shared__ __attribute__((aligned(16))) bf16_t Vt[2][DH * VSTR];
    __shared__ int sh_rng[4][3];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // one-dimensional grid: the query blocks of one (batch, head) run on one XCD, one after another,
    // so that head's K and V are fetched into that XCD's L2 once and then re-read from it
    const int nqb = (a.L + AQ - 1) / AQ;
    const int work = xcd_linear(blockIdx.x, gridDim.x);
    int qb, bh;
    if constexpr (MASKED) {
        // Under a pattern the query blocks differ in work (causal: block qb sees qb + 1 blocks of
        // keys).  The (batch, head) pairs go in groups of hgroup, about one XCD's worth of resident
        // workgroups; inside a group the heaviest query blocks are dispatched first, so the long
        // ones do not start last and form the tail.  K and V of a group stay within one XCD's L2.
        const int nbh = a.H * a.B;
        const int gsz = a.hgroup * nqb;
        const int g = work / gsz, r = work - g * gsz;
        const int gn = min(a.hgroup, nbh - g * a.hgroup);
        qb = nqb - 1 - r / gn;
        bh = g * a.hgroup + r % gn;
    } else {
        qb = work % nqb;
        bh = work / nqb;
    }
    const int h = bh % a.H, b = bh / a.H;
    const int L = a.L, d = a.d;
    const bf16_t* base = (const bf16_t*)a.qkv + (int64_t)b * L * a.ld;
    const int q0 = qb * AQ + wave * 32;
    const int qi = q0 + (lane & 31);
    const int grp = lane >> 5;

    bf16x8 qf[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        if (qi < L) qf[kk] = *(const bf16x8*)(base + (int64_t)qi * a.ld + h * DH + kk * 16 + grp * 8);
        else
#pragma unroll
            for (int e = 0; e < 8; ++e) qf[kk][e] = (__bf16)0.0f;
    }

    f32x16 o[2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[i][e] = 0.f;
    float mrow = -INFINITY, lpart = 0.f;

    // Key tiles of this workgroup: 0 .. ntiles-1, or under a pattern the prefix tiles [0, tp) then
    // the window tiles [tw0, tw1).  Per wavefront: the union bounds (pmax, wlo, whi) decide whether
    // it has work in a tile; the intersection bounds (pmin, lomax, himin) whether the tile is whole.
    int qpre = 0, qlo = 0, qhi = 0;
    int tp = (L + AK - 1) / AK, tw0 = tp, tw1 = tp;
    int pmax = L, wlo = 0, whi = 0, pmin = L, lomax = 0, himin = 0;
    if constexpr (MASKED) {
        if (qi < L) query_window(a, qi, qpre, qlo, qhi);
        const bool win = qhi > qlo;
        pmax = wave_max_i(qpre);
        wlo = wave_min_i(win ? qlo : INT_MAX);
        whi = wave_max_i(win ? qhi : 0);
        // padded queries (qi >= L) see nothing and take no part in the intersection
        pmin = wave_min_i(qi < L ? qpre : INT_MAX);
        lomax = wave_max_i(qi < L ? qlo : INT_MIN);
        himin = wave_min_i(qi < L ? qhi : INT_MAX);
        if (lane == 0) {
            sh_rng[wave][0] = pmax;
            sh_rng[wave][1] = wlo;
            sh_rng[wave][2] = whi;
        }
        __syncthreads();
        int gp = 0, glo = INT_MAX, ghi = 0;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            gp = max(gp, sh_rng[w][0]);
            glo = min(glo, sh_rng[w][1]);
            ghi = max(ghi, sh_rng[w][2]);
        }
        tp = (gp + AK - 1) / AK;
        if (ghi > glo) {
            tw0 = max(tp, glo / AK);
            tw1 = max(tw0, (ghi + AK - 1) / AK);
        } else {
            tw0 = tw1 = tp;
        }
    }
    const int ntiles = tp + (tw1 - tw0);
    auto tile_of = [&](int k) { return k < tp ? k : tw0 + (k - tp); };

    // K tile: thread handles 16-byte chunks c = tid + 256 r (key c / 8, columns 8 (c % 8) ..).
    // V tile (stored transposed): thread handles dv chunk vc = tid / 32 and the pair of keys that
    // sit at transposed positions 2 vp, 2 vp + 1 (vp = tid % 32); these are adjacent keys, so each
    // dv row receives one 32-bit word per thread (a half-wave writes 128 contiguous bytes).
    const int vc = tid >> 5, vp = tid & 31;
    const int vkey = 16 * (vp >> 3) + 4 * ((vp >> 2) & 1) + 8 * ((vp >> 1) & 1) + 2 * (vp & 1);
    uint4 rk[2], rv[2];
    auto gload = [&](int kb0) {
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int c = tid + 256 * r, key = c >> 3, dc = (c & 7) * 8, t = kb0 + key;
            rk[r] = (t < L) ? *(const uint4*)(base + (int64_t)t * a.ld + d + h * DH + dc)
                            : make_uint4(0u, 0u, 0u, 0u);
            const int tv = kb0 + vkey + r;
            rv[r] = (tv < L) ? *(const uint4*)(base + (int64_t)tv * a.ld + 2 * d + h * DH + 8 * vc)
                             : make_uint4(0u, 0u, 0u, 0u);
        }
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int c = tid + 256 * r, key = c >> 3, dc = (c & 7) * 8;
            *(uint4*)&Ks[buf][key * KSTR + dc] = rk[r];
        }
        const uint32_t a0[4] = {rv[0].x, rv[0].y, rv[0].z, rv[0].w};
        const uint32_t a1[4] = {rv[1].x, rv[1].y, rv[1].z, rv[1].w};
        uint32_t wv[8];   // wv[e] = (V[key][8 vc + e], V[key + 1][8 vc + e]) as a bf16 pair
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            wv[2 * e] = __builtin_amdgcn_perm(a1[e], a0[e], 0x05040100u);
            wv[2 * e + 1] = __builtin_amdgcn_perm(a1[e], a0[e], 0x07060302u);
        }
        uint32_t* vt = (uint32_t*)&Vt[buf][0];
#pragma unroll
        for (int e = 0; e < 8; ++e) vt[((8 * vc + e) * VSTR + 2 * vp) >> 1] = wv[e];
    };

    // One 64-key tile.
    // The exponent reference mref is raised only when a row's maximum exceeds it by more than
    // RESCALE (base-2 units), so probabilities stay below 2^RESCALE and the O accumulators are
    // rescaled only on those rare steps (checked once per wavefront).
    constexpr float RESCALE = 8.0f;
    auto tile = [&](int k) {
        const int buf = k & 1, kb0 = tile_of(k) * AK;
        f32x16 sacc[2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
            for (int e = 0; e < 16; ++e) sacc[kb][e] = 0.f;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const bf16x8 kf = *(const bf16x8*)&Ks[buf][(kb * 32 + (lane & 31)) * KSTR + kk * 16 + grp * 8];
                sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], sacc[kb], 0, 0, 0);
            }
        }
        if constexpr (MASKED) {
            // whole tile visible to every query of the wavefront (then also inside L)?
            const bool whole = kb0 + AK <= pmin || (kb0 >= lomax && kb0 + AK <= himin);
            if (!whole) {
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int j = 0; j < 16; ++j) {
                        const int key = kb0 + kb * 32 + 8 * (j >> 2) + 4 * grp + (j & 3);
                        if (!(key < qpre || (key >= qlo && key < qhi))) sacc[kb][j] = -INFINITY;
                    }
            }
        } else if (kb0 + AK > L) {   // wave-uniform: only the last tile can run past L
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    const int key = kb0 + kb * 32 + 8 * (j >> 2) + 4 * grp + (j & 3);
                    if (key >= L) sacc[kb][j] = -INFINITY;
                }
        }
        float mloc = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int j = 0; j < 16; ++j) mloc = fmaxf(mloc, sacc[kb][j]);
        mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64)) * a.scale_log2;
        const bool raise = mloc > mrow + RESCALE;
        if (__any(raise)) {
            const float mnew = raise ? mloc : mrow;
            // a row that has seen no visible key keeps mrow = -inf: its factor must be 1, not NaN
            const float corr = MASKED && !raise ? 1.0f : __builtin_amdgcn_exp2f(mrow - mnew);
            lpart *= corr;
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int e = 0; e < 16; ++e) o[i][e] *= corr;
            mrow = mnew;
        }
        float psum = 0.f;
        const float negm = MASKED && mrow == -INFINITY ? 0.f : -mrow;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const float p = __builtin_amdgcn_exp2f(fmaf(sacc[kb][j], a.scale_log2, negm));
                sacc[kb][j] = p;
                psum += p;
            }
        lpart += psum;
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4) {
            bf16x8 pf;
#pragma unroll
            for (int e = 0; e < 8; ++e) pf[e] = (__bf16)sacc[s4 >> 1][8 * (s4 & 1) + e];
#pragma unroll
            for (int blk = 0; blk < 2; ++blk) {
                const bf16x8 vf = *(const bf16x8*)&Vt[buf][(blk * 32 + (lane & 31)) * VSTR + s4 * 16 + grp * 8];
                o[blk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, o[blk], 0, 0, 0);
            }
        }
    };
    // does any query of this wavefront see a key of the tile starting at kb0?
    auto wave_needs = [&](int kb0) {
        return !MASKED || kb0 < pmax || (kb0 < whi && kb0 + AK > wlo);
    };
    if (ntiles > 0) {
        gload(tile_of(0) * AK);
        sstore(0);
    }
    __syncthreads();
    for (int k = 0; k < ntiles; ++k) {
        if (k + 1 < ntiles) gload(tile_of(k + 1) * AK);
        if (wave_needs(tile_of(k) * AK)) tile(k);
        if (k + 1 < ntiles) sstore((k + 1) & 1);
        __syncthreads();
    }

    const float l = lpart + __shfl_xor(lpart, 32, 64);
    const float inv = 1.0f / l;
    if (qi < L) {
        bf16_t* out = (bf16_t*)a.out + ((int64_t)b * L + qi) * a.ldo + h * DH;
#pragma unroll
        for (int blk = 0; blk < 2; ++blk)
#pragma unroll
            for (int j4 = 0; j4 < 4; ++j4) {
                const int dv = blk * 32 + 8 * j4 + 4 * grp;
                uint2 p;
                p.x = pack_bf16x2(o[blk][4 * j4] * inv, o[blk][4 * j4 + 1] * inv);
                p.y = pack_bf16x2(o[blk][4 * j4 + 2] * inv, o[blk][4 * j4 + 3] * inv);
                *(uint2*)(out + dv) = p;
            }
    }
}

template <int D, bool MASKED>
__global__ __launch_bounds__(128) void attn_f32_kernel(AttnArgs a) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int L = a.L, H = a.H, d = a.d;
    if (idx >= (int64_t)a.B * H * L) return;
    const int q = (int)(idx % L);
    const int h = (int)((idx / L) % H);
    const int b = (int)(idx / ((int64_t)L * H));
    const float* base = (const float*)a.qkv + (int64_t)b * L * a.ld;
    const float scale = 1.0f / sqrtf((float)D);
    float qv[D], acc[D];
#pragma unroll
    for (int c = 0; c < D; ++c) { qv[c] = base[(int64_t)q * a.ld + h * D + c]; acc[c] = 0.f; }
    int pre = L, lo = 0, hi = 0;
    if (MASKED) query_window(a, q, pre, lo, hi);
    float m = -INFINITY, l = 0.f;
    for (int t = 0; t < L; ++t) {
        if (MASKED && !(t < pre || (t >= lo && t < hi))) continue;
        const float* kr = base + (int64_t)t * a.ld + d + h * D;
        float sdot = 0.f;
#pragma unroll
        for (int c = 0; c < D; ++c) sdot = fmaf(qv[c], kr[c], sdot);
        sdot *= scale;
        const float mn = fmaxf(m, sdot);
        const float corr = expf(m - mn), p = expf(sdot - mn);
        l = l * corr + p;
        const float* vr = kr + d;
#pragma unroll
        for (int c = 0; c < D; ++c) acc[c] = fmaf(p, vr[c], acc[c] * corr);
        m = mn;
    }
    float* out = (float*)a.out + ((int64_t)b * L + q) * a.ldo + h * D;
#pragma unroll
    for (int c = 0; c < D; ++c) out[c] = acc[c] / l;
}

bool attn_supported(int dtype, int dh) {
    if (dtype == DD_BF16) return dh == DH;
    return dh == 16 || dh == 32 || dh == 64 || dh == 128;
}

static int num_cus_attn() {
    static int n = 0;
    if (n == 0) {
        int dev = 0, v = 0;
        (void)hipGetDevice(&dev);
        n = (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0) ? v : 256;
    }
    return n;
}

dd_status launch_attn(int dtype, const AttnArgs& a0, hipStream_t s) {
    const int dh = a0.d / a0.H;
    ProfScope ps(KC_ATTN, s);
    AttnArgs a = a0;
    // resident workgroups per XCD (three per CU at the pattern kernel's register count), shared by
    // the query blocks of hgroup (batch, head) pairs
    const int nqb = ceil_div(a.L, AQ);
    a.hgroup = std::max(1, (num_cus_attn() / 8) * 3 / nqb);
    if (dtype == DD_BF16) {
        const dim3 grid((unsigned)(nqb * a.H * a.B));
        if (a.mask) hipLaunchKernelGGL(attn_bf16_kernel<true>, grid, dim3(256), 0, s, a);
        else hipLaunchKernelGGL(attn_bf16_kernel<false>, grid, dim3(256), 0, s, a);
    } else {
        const int64_t n = (int64_t)a.B * a.H * a.L;
        const dim3 grid((unsigned)ceil_div(n, 128));
#define DD_ATTN_F32(DV)                                                                         \
    if (a.mask) hipLaunchKernelGGL((attn_f32_kernel<DV, true>), grid, dim3(128), 0, s, a);      \
    else hipLaunchKernelGGL((attn_f32_kernel<DV, false>), grid, dim3(128), 0, s, a);
        switch (dh) {
            case 16: DD_ATTN_F32(16) break;
            case 32: DD_ATTN_F32(32) break;
            case 64: DD_ATTN_F32(64) break;
            default: DD_ATTN_F32(128) break;
        }
#undef DD_ATTN_F32
    }
    return launch_status("attention");
}

}  // namespace dd
