// Dense layers of the denoiser: C = A W^T (+ epilogue), A [M][K] row-major, W [N][K] row-major
// (weights stored [out][in]), so both operands are contiguous along K.
//
// bf16 path: 128x128x64 workgroup tiles, 4 wavefronts each owning a 64x64 sub-tile computed with
// v_mfma_f32_32x32x16_bf16 (fp32 accumulation).  Global -> register prefetch of the next K-tile
// overlaps the MFMAs on the current one; tiles are double-buffered in padded LDS rows (144 B) so
// the 16-byte fragment reads are bank-conflict free.  The MFMA's first operand is the weight
// fragment, so each lane ends with four consecutive output columns of one row, which the
// epilogue writes as 8-byte (bf16) or 16-byte (fp32 residual) accesses.
//
// Tile order: workgroups are dispatched round-robin over the 8 XCDs; each XCD is given a
// contiguous run of tile ids, walked in groups of 8 M-tiles so concurrent tiles share A and W
// tiles in that XCD's L2.
//
// Epilogues: bias -> bf16 (QKV), bias + GELU(tanh) -> bf16 (MLP up), bias + fp32 residual add in
// place (attention output, MLP down), plain store (vocabulary projection).
#include <math.h>

#include "kernels.h"

namespace dd {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;

// gelu_tanh(x) = 0.5 x (1 + tanh(y)) = x / (1 + exp(-2y)), y = sqrt(2/pi) (x + 0.044715 x^3)
DD_DEV float gelu_tanh(float x) {
    const float y = 0.7978845608028654f * fmaf(0.044715f * x, x * x, x);
    return x / (1.0f + __expf(-2.0f * y));
}

DD_DEV void map_tile(int bid, int nblocks, int tiles_m, int tiles_n, int& tm, int& tn) {
    int t = bid;
    const int per = nblocks / 8;
    if (bid < per * 8) t = (bid & 7) * per + (bid >> 3);
    constexpr int GM = 8;
    const int in_group = GM * tiles_n;
    const int grp = t / in_group;
    const int first = grp * GM;
    const int gsz = min(tiles_m - first, GM);
    const int r = t - grp * in_group;
    tm = first + r % gsz;
    tn = r / gsz;
}

// ------------------------------------------------------------------------------ bf16 MFMA
constexpr int BM = 128, BN = 128, BK = 64, LSTR = BK + 8;

template <int EPI>
DD_DEV void epilogue_bf16(const GemmArgs& g, int m, int n, const float* v) {
    float o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        float x = v[e];
        if (EPI != EPI_PLAIN && n + e < g.N) x += bf16_to_f32(((const bf16_t*)g.bias)[n + e]);
        if (EPI == EPI_BIAS_GELU) x = gelu_tanh(x);
        o[e] = x;
    }
    if (EPI == EPI_BIAS_RESID) {
        float* c = (float*)g.C + (int64_t)m * g.ldc + n;
        if (n + 3 < g.N) {
            float4 h = *(float4*)c;
            h.x += o[0]; h.y += o[1]; h.z += o[2]; h.w += o[3];
            *(float4*)c = h;
        } else {
            for (int e = 0; e < 4; ++e) if (n + e < g.N) c[e] += o[e];
        }
    } else {
        bf16_t* c = (bf16_t*)g.C + (int64_t)m * g.ldc + n;
        if (n + 3 < g.N) {
            uint2 p;
            p.x = pack_bf16x2(o[0], o[1]);
            p.y = pack_bf16x2(o[2], o[3]);
            *(uint2*)c = p;
        } else {
            for (int e = 0; e < 4; ++e) if (n + e < g.N) c[e] = f32_to_bf16(o[e]);
        }
    }
}

template <int EPI>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmArgs g, int tiles_m, int tiles_n) {
    __shared__ __attribute__((aligned(16))) bf16_t As[2][BM * LSTR];
    __shared__ __attribute__((aligned(16))) bf16_t Ws[2][BN * LSTR];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    int tm, tn;
    map_tile(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    const bf16_t* A = (const bf16_t*)g.A;
    const bf16_t* W = (const bf16_t*)g.W;

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    uint4 ra[4], rw[4];
    const int lrow = tid >> 3, lk = (tid & 7) * 8;
    auto gload = [&](int k0) {
        const int gk = k0 + lk;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = lrow + 32 * r;
            const int gm = m0 + row, gn = n0 + row;
            ra[r] = (gm < g.M && gk < g.K) ? *(const uint4*)(A + (int64_t)gm * g.lda + gk)
                                           : make_uint4(0u, 0u, 0u, 0u);
            rw[r] = (gn < g.N && gk < g.K) ? *(const uint4*)(W + (int64_t)gn * g.ldw + gk)
                                           : make_uint4(0u, 0u, 0u, 0u);
        }
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = lrow + 32 * r;
            *(uint4*)&As[buf][row * LSTR + lk] = ra[r];
            *(uint4*)&Ws[buf][row * LSTR + lk] = rw[r];
        }
    };
    auto compute = [&](int buf) {
#pragma unroll
        for (int kk = 0; kk < BK / 16; ++kk) {
            const int koff = kk * 16 + (lane >> 5) * 8;
            bf16x8 af[2], wf[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                af[i] = *(const bf16x8*)&As[buf][(wm * 64 + i * 32 + (lane & 31)) * LSTR + koff];
                wf[i] = *(const bf16x8*)&Ws[buf][(wn * 64 + i * 32 + (lane & 31)) * LSTR + koff];
            }
#pragma unroll
            for (int nb = 0; nb < 2; ++nb)
#pragma unroll
                for (int mb = 0; mb < 2; ++mb)
                    acc[nb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[nb], af[mb], acc[nb][mb], 0, 0, 0);
        }
    };

    const int nk = (g.K + BK - 1) / BK;
    gload(0);
    sstore(0);
    __syncthreads();
    for (int t = 0; t < nk; ++t) {
        if (t + 1 < nk) gload((t + 1) * BK);
        compute(t & 1);
        if (t + 1 < nk) sstore((t + 1) & 1);
        __syncthreads();
    }

#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
            const int m = m0 + wm * 64 + mb * 32 + (lane & 31);
            if (m >= g.M) continue;
#pragma unroll
            for (int j4 = 0; j4 < 4; ++j4) {
                const int n = n0 + wn * 64 + nb * 32 + 8 * j4 + 4 * (lane >> 5);
                if (n >= g.N) continue;
                float v[4] = {acc[nb][mb][4 * j4], acc[nb][mb][4 * j4 + 1], acc[nb][mb][4 * j4 + 2],
                              acc[nb][mb][4 * j4 + 3]};
                epilogue_bf16<EPI>(g, m, n, v);
            }
        }
}

// ------------------------------------------------------------------------------ fp32 (validation)
constexpr int FT = 64, FK = 16;

template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs g, int tiles_m, int tiles_n) {
    __shared__ float As[FK][FT + 4];
    __shared__ float Ws[FK][FT + 4];
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
    const int m0 = tm * FT, n0 = tn * FT;
    const float* A = (const float*)g.A;
    const float* W = (const float*)g.W;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < g.K; k0 += FK) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int idx = tid + 256 * r, row = idx / FK, k = idx % FK;
            const int gk = k0 + k;
            As[k][row] = (m0 + row < g.M && gk < g.K) ? A[(int64_t)(m0 + row) * g.lda + gk] : 0.f;
            Ws[k][row] = (n0 + row < g.N && gk < g.K) ? W[(int64_t)(n0 + row) * g.ldw + gk] : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < FK; ++k) {
            float a[4], w[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) { a[i] = As[k][ty * 4 + i]; w[i] = Ws[k][tx * 4 + i]; }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], w[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int m = m0 + ty * 4 + i;
        if (m >= g.M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int n = n0 + tx * 4 + j;
            if (n >= g.N) continue;
            float x = acc[i][j];
            if (EPI != EPI_PLAIN) x += ((const float*)g.bias)[n];
            if (EPI == EPI_BIAS_GELU) x = 0.5f * x * (1.0f + tanhf(0.7978845608028654f * (x + 0.044715f * x * x * x)));
            float* c = (float*)g.C + (int64_t)m * g.ldc + n;
            if (EPI == EPI_BIAS_RESID) *c += x;
            else *c = x;
        }
    }
}

template <int EPI>
static void launch_epi(int dtype, const GemmArgs& g, hipStream_t s) {
    if (dtype == DD_BF16) {
        const int tm = (g.M + BM - 1) / BM, tn = (g.N + BN - 1) / BN;
        hipLaunchKernelGGL(gemm_bf16_kernel<EPI>, dim3(tm * tn), dim3(256), 0, s, g, tm, tn);
    } else {
        const int tm = (g.M + FT - 1) / FT, tn = (g.N + FT - 1) / FT;
        hipLaunchKernelGGL(gemm_f32_kernel<EPI>, dim3(tm * tn), dim3(256), 0, s, g, tm, tn);
    }
}

dd_status launch_gemm(int dtype, int epi, int cls, const GemmArgs& g, hipStream_t s) {
    if (g.M == 0 || g.N == 0) return DD_OK;
    ProfScope ps(cls, s);
    switch (epi) {
        case EPI_BIAS: launch_epi<EPI_BIAS>(dtype, g, s); break;
        case EPI_BIAS_GELU: launch_epi<EPI_BIAS_GELU>(dtype, g, s); break;
        case EPI_BIAS_RESID: launch_epi<EPI_BIAS_RESID>(dtype, g, s); break;
        default: launch_epi<EPI_PLAIN>(dtype, g, s); break;
    }
    return launch_status("gemm");
}

}  // namespace dd
