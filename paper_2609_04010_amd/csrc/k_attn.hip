// Multi-head attention softmax(q k^T / sqrt(dh)) v, flash style (no L x L tensor), over every key
// or, with a visibility pattern, over the keys j of query i with j < pre_i or lo_i <= j < hi_i (a
// prefix plus one window: bidirectional, causal, block-causal and the [x, z_1] block-diffusion
// pattern all take this form).
//
// bf16 path (dh = 64): a workgroup of 4 wavefronts owns 128 queries of one (batch, head); each
// wavefront owns 32 queries.  Key/value tiles of 64 tokens go global -> LDS directly
// (global_load_lds_dwordx4, double-buffered, no staging registers, which leaves room for four
// wavefronts per SIMD), K and V both row-major in 128-byte rows whose 16-byte chunks are
// XOR-swizzled by row; the P.V contraction reads its V^T operand with gfx950's transposing LDS
// read (ds_read_b64_tr_b16).
//   S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (first operand: K rows from LDS; second: the wave's
//         Q fragment, held in registers for the whole kernel).  Each lane then holds 32 scores of
//         one query, the other 32 of the tile being in lane ^ 32.
//   Online softmax in base 2 with the 1/sqrt(dh) scale folded into the exponent.  The exponent
//         reference is the row maximum of the first tile (one cross-lane exchange) and stays while
//         the probabilities of later tiles remain below 2^64; only a tile that exceeds that takes
//         its maximum again and raises the reference.  The running sum stays per lane until the end.
//   O^T += V^T P^T: the probabilities are rounded to bf16 and used directly as the second MFMA
//         operand (no shuffles), so each lane's output column is again its own query.  The first
//         operand needs, per lane, one head column of V at the 8 keys the accumulator layout of S^T
//         gives that lane's probabilities: two transposing reads of 4 consecutive keys each.
// Patterns (MASKED instance): a workgroup visits only the key tiles that meet the union of its
// queries' visible sets (the prefix tiles, then the window tiles); a wavefront whose queries see
// nothing of a tile skips its arithmetic; a tile that every query of the wavefront sees whole takes
// no per-element test.  Rows that have seen no visible key yet keep mref = -inf and use exponent
// reference 0, so their probabilities are exactly 0 until their first visible key.
// fp32 path (validation): one thread per (batch, head, query), fp32 online softmax.
#include <limits.h>
#include <math.h>

#include <algorithm>
#include <type_traits>

#include "kernels.h"

namespace dd {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;

constexpr int AQ = 128;  // queries per workgroup
constexpr int AK = 64;   // keys per tile
constexpr int DH = 64;
constexpr int KROW = DH;   // bf16 per LDS row (128 bytes, no padding: chunks are swizzled)

typedef short v4s __attribute__((ext_vector_type(4)));
typedef short v8s __attribute__((ext_vector_type(8)));

// ds_read_b64_tr_b16 (gfx950): in each group of 16 lanes the 16 addresses name a 16 x 4 matrix M of
// 16-bit elements (row j: the 4 elements at lane j's address); lane i receives M[4e + i/4][i % 4],
// e = 0..3.  With lane j of the group pointing at V[k0 + j / 4][c0 + 4 (j % 4)] (row-major V), lane i
// receives V[k0 + e][c0 + i]: four consecutive keys of head column c0 + i.
//
// LDS rows are 128 bytes (one key, 64 head columns); even rows fill banks 0-31, odd rows 32-63.
// 16-byte chunk c of row r sits at slot c ^ sw(r):
//   K: sw(r) = (r >> 1) & 7 -- a fragment read (16 lanes: rows r0..r0+15, one chunk) meets 8
//      different slots in each bank half;
//   V: sw(r) = r & 6 -- a transposing read (16 lanes: rows k..k+3, k % 4 == 0, two adjacent chunks
//      x, x ^ 1 per row) gives rows k and k + 2 the slot pairs {x, x ^ 1} and {x ^ 2, x ^ 3}.
DD_DEV int ksw(int r) { return (r >> 1) & 7; }
DD_DEV int vsw(int r) { return r & 6; }

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void gbl_void;
DD_DEV v4s ds_read_tr16(const bf16_t* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s*)p);
}

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

template <bool MASKED, bool LISTED = false>
__global__ __launch_bounds__(256, MASKED ? 3 : 4) void attn_bf16_kernel(AttnArgs a) {
    __shared__ __attribute__((aligned(1024))) bf16_t Ks[2][AK * KROW];
    __shared__ __attribute__((aligned(1024))) bf16_t Vs[2][AK * KROW];
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
    int qi = q0 + (lane & 31);
    const int grp = lane >> 5;
    if constexpr (LISTED) {
        // query block qb of sequence b's listed rows; qi becomes the position of this lane's query
        // (L: none).  The test is the same for the whole workgroup, so it leaves before any barrier.
        const int s0 = a.qseq[b], s1 = a.qseq[b + 1];
        if (s0 + qb * AQ >= s1) return;
        qi = s0 + qi < s1 ? a.qrows[s0 + qi] - b * L : L;
    }

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

    // Tile loads: 8 KB of K and 8 KB of V per tile, eight 1 KB wave instructions each; wavefront w
    // issues K and V instructions 2w and 2w + 1 (rows 8 i .. 8 i + 7).  Lane l fills LDS slot l % 8 of
    // row 8 i + l / 8 with the global chunk that belongs there.  Keys past L read row L - 1 (their
    // scores are masked to -inf, so their probabilities are exactly 0).
    // Per-lane offsets (elements from the tile's first key row, under 64 rows of the qkv matrix, so
    // well inside 32 bits) are fixed; a tile adds kb0 rows.  The ragged last tile (rows past L read
    // row L - 1) takes a separate, scalar-branched path.
    const int sl = lane & 7;
    int ok[2], ov[2];
#pragma unroll
    for (int ii = 0; ii < 2; ++ii) {
        const int r = 8 * (2 * wave + ii) + (lane >> 3);
        ok[ii] = r * (int)a.ld + d + h * DH + 8 * (sl ^ ksw(r));
        ov[ii] = r * (int)a.ld + 2 * d + h * DH + 8 * (sl ^ vsw(r));
    }
    auto dma = [&](int kb0, int buf) {
        const bf16_t* tb = base + (int64_t)kb0 * a.ld;
        if (kb0 + AK <= L) {
#pragma unroll
            for (int ii = 0; ii < 2; ++ii) {
                const int i = 2 * wave + ii;
                __builtin_amdgcn_global_load_lds((gbl_void*)(tb + ok[ii]), (lds_void*)&Ks[buf][8 * i * KROW], 16, 0, 0);
                __builtin_amdgcn_global_load_lds((gbl_void*)(tb + ov[ii]), (lds_void*)&Vs[buf][8 * i * KROW], 16, 0, 0);
            }
        } else {
#pragma unroll
            for (int ii = 0; ii < 2; ++ii) {
                const int i = 2 * wave + ii, r = 8 * i + (lane >> 3);
                const bf16_t* row = tb + (int64_t)min(r, L - 1 - kb0) * a.ld + h * DH;
                __builtin_amdgcn_global_load_lds((gbl_void*)(row + d + 8 * (sl ^ ksw(r))),
                                                 (lds_void*)&Ks[buf][8 * i * KROW], 16, 0, 0);
                __builtin_amdgcn_global_load_lds((gbl_void*)(row + 2 * d + 8 * (sl ^ vsw(r))),
                                                 (lds_void*)&Vs[buf][8 * i * KROW], 16, 0, 0);
            }
        }
    };

    // The exponent reference mref is raised only when a row's maximum exceeds it by more than
    // RESCALE (base-2 units), so probabilities stay below 2^RESCALE and the O accumulators are
    // rescaled only on those rare steps (checked once per wavefront).
    constexpr float RESCALE = 8.0f;
    // One 64-key tile; `part`: the tile is not entirely visible to every query of the wavefront
    // (the ragged last tile, or pattern boundaries), so scores get the per-element key test.
    auto tile = [&](int k, bool part) {
        const int buf = k & 1, kb0 = tile_of(k) * AK;
        f32x16 sacc[2];
        // The MFMA blocks (QK^T here, PV below) run at wave priority 1, so that of the four
        // wavefronts of a SIMD the one with MFMAs to issue goes first and the softmax VALU work
        // of the others fills in (62.1-62.5 vs 62.9-63.6 us at B16 L1024; priority on the
        // exponentials instead: 64.7 us)
        auto scores = [&]() {
            __builtin_amdgcn_s_setprio(1);
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
                for (int e = 0; e < 16; ++e) sacc[kb][e] = 0.f;
#pragma unroll
                for (int kk = 0; kk < 4; ++kk) {
                    const int kr = kb * 32 + (lane & 31);
                    const bf16x8 kf = *(const bf16x8*)&Ks[buf][kr * KROW + 8 * ((2 * kk + grp) ^ ksw(kr))];
                    sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], sacc[kb], 0, 0, 0);
                }
            }
            __builtin_amdgcn_s_setprio(0);
            if (part) {
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int j = 0; j < 16; ++j) {
                        const int key = kb0 + kb * 32 + 8 * (j >> 2) + 4 * grp + (j & 3);
                        const bool vis = MASKED ? (key < qpre || (key >= qlo && key < qhi)) : key < L;
                        if (!vis) sacc[kb][j] = -INFINITY;
                    }
            }
        };
        auto exps = [&](float negm) {
            float ps = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    const float p = __builtin_amdgcn_exp2f(fmaf(sacc[kb][j], a.scale_log2, negm));
                    sacc[kb][j] = p;
                    ps += p;
                }
            return ps;
        };
        scores();
        float psum = 0.f;
        bool done = false;
        // Once every row of the wavefront has an exponent reference it usually stays where it is:
        // probabilities up to 2^64 are harmless in fp32 and bf16, so the tile maximum is not needed
        // unless a lane's sum exceeds that (or is not a number).  Then the scores are computed again
        // and the tile takes the path below.
        if (!__any(mrow == -INFINITY)) {
            psum = exps(-mrow);
            done = !__any(!(psum <= 0x1p64f));
            if (!done) {
                asm volatile("");
                scores();
            }
        }
        if (!done) {
            float mloc = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int j = 0; j < 16; ++j) mloc = fmaxf(mloc, sacc[kb][j]);
            mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64)) * a.scale_log2;
            const bool raise = mloc > mrow + RESCALE;
            if (__any(raise)) {
                // rare after the first tile: kept a real branch (an empty volatile asm stops the
                // compiler from executing the 33 multiplies below unconditionally)
                asm volatile("");
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
            psum = exps(MASKED && mrow == -INFINITY ? 0.f : -mrow);
        }
        lpart += psum;
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4) {
            bf16x8 pf;
#pragma unroll
            for (int e = 0; e < 8; ++e) pf[e] = (__bf16)sacc[s4 >> 1][8 * (s4 & 1) + e];
            // this lane's 8 operand keys: 4 grp + {0..3} and 8 + 4 grp + {0..3} within the step's 16
            const int vk = (s4 >> 1) * 32 + 16 * (s4 & 1) + 4 * grp + ((lane & 15) >> 2);
#pragma unroll
            for (int blk = 0; blk < 2; ++blk) {
                // column blk 32 + 16 ((lane >> 4) & 1) + 4 (lane & 3): chunk vc, half vh
                const int vc = 4 * blk + 2 * ((lane >> 4) & 1) + ((lane >> 1) & 1), vh = 4 * (lane & 1);
                const v4s lo = ds_read_tr16(&Vs[buf][vk * KROW + 8 * (vc ^ vsw(vk)) + vh]);
                const v4s hi = ds_read_tr16(&Vs[buf][(vk + 8) * KROW + 8 * (vc ^ vsw(vk + 8)) + vh]);
                const v8s v8 = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                const bf16x8 vf = __builtin_bit_cast(bf16x8, v8);
                o[blk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, o[blk], 0, 0, 0);
            }
        }
        __builtin_amdgcn_s_setprio(0);
    };
    // does any query of this wavefront see a key of the tile starting at kb0?
    auto wave_needs = [&](int kb0) {
        return !MASKED || kb0 < pmax || (kb0 < whi && kb0 + AK > wlo);
    };
    // tile k + 1 streams into the other buffer while tile k is computed; that buffer was last
    // read in tile k - 1, which every wavefront finished before the barrier ending it
    if (ntiles > 0) dma(tile_of(0) * AK, 0);
    __builtin_amdgcn_s_waitcnt(0x3F70);          // vmcnt(0)
    __syncthreads();
    for (int k = 0; k < ntiles; ++k) {
        // the next tile's loads go out at the top wave priority, ahead of the MFMA and softmax
        // work of the SIMD's other wavefronts (61.5-62.2 vs 63.2-65.2 us at B16 L1024)
        __builtin_amdgcn_s_setprio(3);
        if (k + 1 < ntiles) dma(tile_of(k + 1) * AK, (k + 1) & 1);
        __builtin_amdgcn_s_setprio(0);
        const int kb0 = tile_of(k) * AK;
        // is the tile entirely visible to every query of this wavefront (and inside L)?
        const bool whole = MASKED ? (kb0 + AK <= pmin || (kb0 >= lomax && kb0 + AK <= himin)) : kb0 + AK <= L;
        if (wave_needs(kb0)) tile(k, !whole);
        __builtin_amdgcn_s_waitcnt(0x3F70);      // vmcnt(0): this lane's loads of tile k + 1 landed
        __syncthreads();                          // ... everyone's
    }

    const float l = lpart + __shfl_xor(lpart, 32, 64);
    const float inv = 1.0f / l;
    if (qi < L) {
        // listed queries are written in list order
        const int64_t orow = LISTED ? (int64_t)a.qseq[b] + q0 + (lane & 31) : (int64_t)b * L + qi;
        bf16_t* out = (bf16_t*)a.out + orow * a.ldo + h * DH;
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
    if (a.qrows && (dtype != DD_BF16 || a.mask || !a.qseq)) {
        set_error("listed queries need the bf16 path, no pattern and the sequence starts");
        return DD_E_UNSUPPORTED;
    }
    if (dtype == DD_BF16) {
        const dim3 grid((unsigned)(nqb * a.H * a.B));
        if (a.mask) launch_k(attn_bf16_kernel<true>, grid, dim3(256), 0, s, a);
        else if (a.qrows) launch_k((attn_bf16_kernel<false, true>), grid, dim3(256), 0, s, a);
        else launch_k(attn_bf16_kernel<false>, grid, dim3(256), 0, s, a);
    } else {
        const int64_t n = (int64_t)a.B * a.H * a.L;
        const dim3 grid((unsigned)ceil_div(n, 128));
#define DD_ATTN_F32(DV)                                                                         \
    if (a.mask) launch_k((attn_f32_kernel<DV, true>), grid, dim3(128), 0, s, a);      \
    else launch_k((attn_f32_kernel<DV, false>), grid, dim3(128), 0, s, a);
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
