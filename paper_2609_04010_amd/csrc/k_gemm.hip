// Dense layers of the denoiser: C = A W^T (+ epilogue), A [M][K] row-major, W [N][K] row-major
// (weights stored [out][in]), so both operands are contiguous along K.
//
// bf16 path: workgroup tiles of 128 or 256 rows/columns by 64 along K, 4 wavefronts each owning a
// quarter of the tile, computed with v_mfma_f32_32x32x16_bf16 (fp32 accumulation).  Global -> register prefetch of the next K-tile
// overlaps the MFMAs on the current one; tiles are double-buffered in padded LDS rows (144 B) so
// the 16-byte fragment reads are bank-conflict free.  The MFMA's first operand is the weight
// fragment, so each lane ends with four consecutive output columns of one row, which the
// epilogue writes as 8-byte (bf16) or 16-byte (fp32 residual) accesses.
//
// Tile order: workgroups are dispatched round-robin over the 8 XCDs; each XCD is given a
// contiguous run of tile ids, walked in groups of 8 M-tiles so concurrent tiles share A and W
// tiles in that XCD's L2.
//
// bf16 outputs other than QKV's are written with non-temporal stores: they are read by the next
// kernel, not by this one, so they should not push the operand tiles other workgroups still reuse
// out of L2 (measured: MLP up 91 -> 85 us at B16 L1024).  The QKV output and the fp32 residual row
// are stored normally (see the epilogues).
//
// Epilogues: bias -> bf16 (QKV), bias + GELU(tanh) -> bf16 (MLP up), bias + fp32 residual add in
// place (attention output, MLP down), plain store (vocabulary projection), plain store plus the
// per-row log-sum-exp of each 256-column group (vocabulary projection feeding the sampler), per-row
// gate x scale -> bf16 (adapter down-projection of a gated LoRA).
#include <math.h>
#include <stdlib.h>

#include <algorithm>
#include <type_traits>

#include "kernels.h"
#include "rng.h"

namespace dd {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(4))) float f32x4;

// gelu_tanh(x) = 0.5 x (1 + tanh(y)) = x / (1 + exp(-2y)), y = sqrt(2/pi) (x + 0.044715 x^3), with
// exp(-2y) = 2^(x (a + b x^2)), a = -2 sqrt(2/pi) log2(e), b = 0.044715 a: five VALU operations plus
// v_exp_f32 and v_rcp_f32 (about 1 ulp each; the result is rounded to bf16 afterwards)
DD_DEV float gelu_tanh(float x) {
    const float e = __builtin_amdgcn_exp2f(x * fmaf(x * x, -0.1029432395800235f, -2.302208198144325f));
    return x * __builtin_amdgcn_rcpf(1.0f + e);
}

// M-tiles per group of the tile order (map_tile) of the body projections other than QKV (4; QKV
// takes 2, the vocabulary projection 8: see the kernel).  Measured: QKV 69.6 -> 66.0 us with 4
// instead of 8, the others unchanged; the vocabulary projection slower with 4.
#ifndef DD_GEMM_GM_BODY
#define DD_GEMM_GM_BODY 4
#endif
template <int GM = 8>
DD_DEV void map_tile(int bid, int nblocks, int tiles_m, int tiles_n, int& tm, int& tn) {
    const int t = xcd_linear(bid, nblocks);
    const int in_group = GM * tiles_n;
    const int grp = t / in_group;
    const int first = grp * GM;
    const int gsz = min(tiles_m - first, GM);
    const int r = t - grp * in_group;
    tm = first + r % gsz;
    tn = r / gsz;
}

// ------------------------------------------------------------------------------ bf16 MFMA
constexpr int BK = 64, LSTR = BK + 8;
constexpr float LOG2E_F = 1.4426950408889634f;

// x rounded to bf16 (round to nearest even, like the stores), as an fp32 value: one conversion that
// writes bf16(0) to the low and bf16(x) to the high half of the word
DD_DEV float round_bf16(float x) {
    uint32_t r;
    asm("v_cvt_pk_bf16_f32 %0, 0, %1" : "=v"(r) : "v"(x));
    return __uint_as_float(r);
}

// EPI_GATE row factor of output row m (m % gate_period is in range for any m, clamped rows too)
DD_DEV float gate_row_scale(const GemmArgs& g, int m) {
    if (!g.gate) return g.gate_scale;
    return g.gate[m % g.gate_period] != 0 ? g.gate_scale : 0.f;
}

template <int EPI>
DD_DEV void epilogue_bf16(const GemmArgs& g, int m, int n, const float* v, const float* bias4) {
    float o[4];
    const float rs = EPI == EPI_GATE ? gate_row_scale(g, m) : 1.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        float x = v[e] + bias4[e];
        if (EPI == EPI_BIAS_GELU) x = gelu_tanh(x);
        if (EPI == EPI_GATE) x = v[e] * rs;
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

// Workgroup tile TBM x TBN (x BK): 4 wavefronts in a 2 x 2 grid, each owning a (TBM/2) x (TBN/2)
// sub-tile of MB x NB 32x32 MFMA blocks.  Larger wave tiles read fewer LDS bytes per MFMA flop
// (64x64: 32 flop/B, 128x128: 64 flop/B).
template <int TBM, int TBN, int EPI>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmArgs g, int tiles_m, int tiles_n) {
    constexpr int MB = TBM / 64, NB = TBN / 64;       // 32x32 blocks per wave along M and N
    constexpr int RA = TBM / 32, RW = TBN / 32;       // 16-byte chunks per thread per K-tile
    extern __shared__ __attribute__((aligned(16))) bf16_t smem[];
    bf16_t* As = smem;                        // [2][TBM * LSTR]
    bf16_t* Ws = smem + 2 * TBM * LSTR;       // [2][TBN * LSTR]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    int tm, tn;
    map_tile(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
    const int m0 = tm * TBM, n0 = tn * TBN;
    const bf16_t* A = (const bf16_t*)g.A;
    const bf16_t* W = (const bf16_t*)g.W;

    f32x16 acc[NB][MB];
#pragma unroll
    for (int i = 0; i < NB; ++i)
#pragma unroll
        for (int j = 0; j < MB; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    uint4 ra[RA], rw[RW];
    const int lrow = tid >> 3, lk = (tid & 7) * 8;
    auto gload = [&](int k0) {
        const int gk = k0 + lk;
#pragma unroll
        for (int r = 0; r < RA; ++r) {
            const int gm = m0 + lrow + 32 * r;
            ra[r] = (gm < g.M && gk < g.K) ? *(const uint4*)(A + (int64_t)gm * g.lda + gk)
                                           : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            const int gn = n0 + lrow + 32 * r;
            rw[r] = (gn < g.N && gk < g.K) ? *(const uint4*)(W + (int64_t)gn * g.ldw + gk)
                                           : make_uint4(0u, 0u, 0u, 0u);
        }
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int r = 0; r < RA; ++r)
            *(uint4*)&As[buf * TBM * LSTR + (lrow + 32 * r) * LSTR + lk] = ra[r];
#pragma unroll
        for (int r = 0; r < RW; ++r)
            *(uint4*)&Ws[buf * TBN * LSTR + (lrow + 32 * r) * LSTR + lk] = rw[r];
    };
    auto compute = [&](int buf) {
        const bf16_t* Ab = As + buf * TBM * LSTR + (wm * (TBM / 2) + (lane & 31)) * LSTR;
        const bf16_t* Wb = Ws + buf * TBN * LSTR + (wn * (TBN / 2) + (lane & 31)) * LSTR;
#pragma unroll
        for (int kk = 0; kk < BK / 16; ++kk) {
            const int koff = kk * 16 + (lane >> 5) * 8;
            bf16x8 af[MB], wf[NB];
#pragma unroll
            for (int i = 0; i < MB; ++i) af[i] = *(const bf16x8*)&Ab[i * 32 * LSTR + koff];
#pragma unroll
            for (int i = 0; i < NB; ++i) wf[i] = *(const bf16x8*)&Wb[i * 32 * LSTR + koff];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
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
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int j4 = 0; j4 < 4; ++j4) {
            const int n = n0 + wn * (TBN / 2) + nb * 32 + 8 * j4 + 4 * (lane >> 5);
            if (n >= g.N) continue;
            float b4[4] = {0.f, 0.f, 0.f, 0.f};
            if (EPI != EPI_PLAIN && EPI != EPI_GATE)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (n + e < g.N) b4[e] = bf16_to_f32(((const bf16_t*)g.bias)[n + e]);
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
                const int m = m0 + wm * (TBM / 2) + mb * 32 + (lane & 31);
                if (m >= g.M) continue;
                float v[4] = {acc[nb][mb][4 * j4], acc[nb][mb][4 * j4 + 1], acc[nb][mb][4 * j4 + 2],
                              acc[nb][mb][4 * j4 + 3]};
                epilogue_bf16<EPI>(g, m, n, v, b4);
            }
        }
}

// ------------------------------------------------------------------------------ bf16, direct to LDS
// 256 x TBN x 64 workgroup tile (TBN = 256 or 192) over a WGM x WGN grid of wavefronts (2 x 2 with
// 128 x TBN/2 sub-tiles, or 8 wavefronts: 2 x 4 of 128 x 64 / 4 x 2 of 64 x 96), each sub-tile a set
// of 32x32 MFMA blocks.  Operand tiles travel global -> LDS with global_load_lds_dwordx4 (no
// staging registers): each wave instruction fills 1 KB = 8 rows of 128 B.  The LDS serves a
// 16-byte read for 16 lanes (256 B, 64 banks) per cycle, and a fragment read covers rows r..r+15 of
// one K-chunk, so the eight 16-byte K-chunks of a row are stored XOR-swizzled with
// slot = chunk ^ ((row >> 1) & 7): the eight even and the eight odd rows of the group each land on
// eight different bank groups.  Two LDS stages.  After the barrier that publishes K-tile t, the
// 16-wide K steps of t run their MFMAs with, between them, the fragment reads of the next step and
// (during the first LD_STEPS steps) the global->LDS loads of K-tile t+1: a load waits in the
// vector-memory queue behind the other wavefronts' loads, and with MFMAs already issued ahead of it
// the matrix core keeps working meanwhile.
// bf16 outputs are staged per wave in padded LDS rows and written as 16-byte row segments.
// The 192-wide variant exists for tile quantisation: with d = 768 it divides N = 768, 2304 and
// 3072 into whole rounds of 256 CUs.  Requires K % 128 == 0; rows past M or N are clamped (their
// results are never stored).
constexpr int DM = 256;                       // tile rows (M) of the wide tiles
// DM_ x TBN_ tiles over WGM x WGN wavefronts, each owning a WM x WN sub-tile of MB x NB 32x32 MFMA
// blocks.  The 64-row form (64 x 128, four wavefronts side by side) serves skinny products: every
// CU streams one 64-row strip of A while all of them share the small W through L2.
template <int TBN_, int WGM_, int WGN_, int DM_ = DM> struct DLShape {
    static constexpr int DM = DM_;                            // tile rows (M)
    static constexpr int TBN = TBN_;                          // tile columns (N)
    static constexpr int WGM = WGM_, WGN = WGN_, NW = WGM * WGN;
    static constexpr int THREADS = 64 * NW;
    static constexpr int WM = DM / WGM, WN = TBN / WGN;       // wave sub-tile
    static constexpr int MB = WM / 32, NB = WN / 32;
    static constexpr int ALOADS = DM / 8 / NW;                // A load instructions per wave per stage
    static constexpr int WLOADS = TBN / 8 / NW;               // W load instructions per wave per stage
    static constexpr int STAGE = (DM + TBN) * BK;             // bf16 elements per stage
    static constexpr int CSTR = WN + 8;                       // epilogue staging row stride (bf16)
    // two operand stages; the epilogue stages half a sub-tile per wave above stage 0
    static constexpr size_t STAGING = (size_t)STAGE * 2 + (size_t)NW * (WM / 2) * CSTR * 2;
    static constexpr size_t LDS = STAGING > (size_t)2 * STAGE * 2 ? STAGING : (size_t)2 * STAGE * 2;
    // workgroups per CU the launcher allows: one for the wide tiles (persistent), several for the
    // one-wavefront skinny tile, whose K loop is latency-bound
    static constexpr int WG_PER_CU = NW >= 4 ? 1 : 8 / NW;
    static_assert(WM % 64 == 0 && WN % 32 == 0 && (MB * NB) % 2 == 0, "wave sub-tile (two row halves)");
    static_assert(DM % (8 * NW) == 0 && TBN % (8 * NW) == 0, "load split");
    static_assert(LDS <= 160 * 1024, "LDS");
};

#ifndef DD_GEMM_RING
#define DD_GEMM_RING 1
#endif
// Operand ring of the residual projections (attention output, MLP down) on the 256 x 192 tile
// (eight wavefronts): A in three LDS stages and W in two, so that A's K-tile G + 2 and W's K-tile
// G + 1 stream in while K-tile G is computed.  A is the operand that mostly comes from HBM (each A
// strip is read by the four tiles across N = d, W by every tile of the XCD), and with one K-tile of
// lead the loop waited for its loads.  The other projections (QKV, MLP up) gained nothing from it.
template <int EPI, class S> constexpr bool dl_ring() {
    return DD_GEMM_RING && S::TBN == 192 && S::DM == 256 && S::NW == 8 && EPI == EPI_BIAS_RESID;
}
// the ring's LDS: three A stages and two W stages (the residual epilogue stages in the A stage of
// the last K-tile)
template <class S> constexpr size_t dl_ring_lds() {
    return ((size_t)3 * S::DM * BK + (size_t)2 * S::TBN * BK) * sizeof(bf16_t);
}

// LDS of the direct-to-LDS kernel: the shape's stages and staging (or the ring's), plus for EPI_LSE
// the (max, sum) partials of each tile row from each of the WGN wavefronts across it
template <int EPI, class S> constexpr size_t dl_lds_bytes() {
    if constexpr (dl_ring<EPI, S>()) return dl_ring_lds<S>();
    return S::LDS + (EPI == EPI_LSE || EPI == EPI_LSE_CDF ? (size_t)S::DM * S::WGN * sizeof(float2) : 0) +
           (EPI == EPI_LSE_CDF ? (size_t)S::DM * sizeof(float2) : 0);
}

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void gbl_void;

// ROLE (the profiler class of the layer) only separates the symbols of layers sharing an epilogue.
// Persistent: workgroup b takes tiles b, b + G, b + 2G, ... (G = grid size).  The number of K-tiles
// is even, so the loads of the next tile's first K-tile go out during the last K-tile of the
// current one into stage 0, which the staged epilogue leaves alone: they land while it runs.  (The
// operand ring of the residual projections fetches the next tile's first K-tiles the same way, into
// the stages its epilogue does not use.)
template <int EPI, int ROLE, int TBN_, int WGM_, int WGN_, int DM_>
__global__ __launch_bounds__(64 * WGM_ * WGN_, 1) void gemm_bf16_dl_kernel(GemmArgs g, int tiles_m, int tiles_n) {
    using S = DLShape<TBN_, WGM_, WGN_, DM_>;
    constexpr int DM = S::DM;
    constexpr int MB = S::MB, NB = S::NB, NA = S::ALOADS, NWL = S::WLOADS;
    constexpr bool GROUP_EPI = EPI == EPI_LSE || EPI == EPI_LSE_CDF;
    // M-tiles per group of the tile order: 8 for the vocabulary projection, 2 for QKV (whose output,
    // stored normally, shares L2 with the operand tiles: 63.3-64.0 -> 60.3-60.7 us with 2 instead of
    // 4 at B16 L1024), 4 for the other body projections
    constexpr int TILE_GM = (EPI == EPI_PLAIN || GROUP_EPI) ? 8 : (EPI == EPI_BIAS ? 2 : DD_GEMM_GM_BODY);
    constexpr int AROWS = DM / S::NW, WROWS = S::TBN / S::NW;   // operand rows each wave loads
    constexpr bool RING = dl_ring<EPI, S>();
    constexpr int AST = DM * BK, WST = S::TBN * BK;   // elements of one ring stage of A / W
    static_assert(!RING || (NA < 16 && dl_ring_lds<S>() <= 160 * 1024 && S::NW * 32 * 32 * 2 <= AST),
                  "ring: the wait counts A's loads, and one A stage holds the residual staging");
    extern __shared__ __attribute__((aligned(1024))) bf16_t smem[];
    // the LDS of A's and W's K-tile G (G counts K-tiles over the workgroup's tiles; nk is even, so
    // without the ring G & 1 is also the tile's own K-tile parity)
    auto a_stage = [&](int G) -> bf16_t* { return RING ? smem + (G % 3) * AST : smem + (G & 1) * S::STAGE; };
    auto w_stage = [&](int G) -> bf16_t* {
        return RING ? smem + 3 * AST + (G & 1) * WST : smem + (G & 1) * S::STAGE + DM * BK;
    };
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / S::WGN, wn = wave % S::WGN;
    // Gathered mode: only the first *m_count output rows exist; the tile grid is re-derived from
    // that device-side count.
    int M = g.M;
    if (g.m_count) {
        M = *g.m_count;
        tiles_m = (M + DM - 1) / DM;
        if (g.m_gate > 0 && ((M > g.m_gate) == (g.m_side != 0))) return;   // the other launch's rows
    }
    const int nblocks = tiles_m * tiles_n;
    int L = blockIdx.x;
    if (L >= nblocks) return;
    const bf16_t* A = (const bf16_t*)g.A;
    const bf16_t* W = (const bf16_t*)g.W;
    const int nk = g.K / BK;                     // even (the launcher checks K % 128 == 0)

    // this lane's source rows: wave w fills A rows AROWS w + 8 i + lane / 8 and W rows
    // WROWS w + 8 i + lane / 8; its 16-byte slot lane % 8 holds K-chunk (lane % 8) ^ ((row >> 1) & 7)
    auto lchunk = [&](int row) { return (lane & 7) ^ ((row >> 1) & 7); };
    // K order of a tile: K-tile t reads K-slice (t + skew) mod nk.  For the vocabulary projection
    // the workgroups that share an operand tile (the 8 M-tiles of a group share W, the N-tiles of
    // one M-tile share A) start at different K-slices, so they do not request the same L2 lines
    // at the same moment (measured 8 % on that GEMM; the accumulation order is all that changes).
    int m0 = 0, n0 = 0, skew = 0;
    // this tile's operand offsets, and (ring) the next tile's, which the last K-tiles fetch from
    int64_t offA[NA], offW[NWL], offAn[RING ? NA : 1], offWn[RING ? NWL : 1];
    auto a_offsets = [&](int tm0, int64_t* o) {
#pragma unroll
        for (int i = 0; i < NA; ++i) {
            const int rl = AROWS * wave + 8 * i + (lane >> 3);
            const int r = min(tm0 + rl, M - 1);
            // (the ring reads the next tile's offsets inside the K loop, where a gathered row id
            // would be a global load to wait for; its launcher never passes a_rows)
            o[i] = (int64_t)(!RING && g.a_rows ? g.a_rows[r] : r) * g.lda + lchunk(rl) * 8;
        }
    };
    auto w_offsets = [&](int tn0, int64_t* o) {
#pragma unroll
        for (int i = 0; i < NWL; ++i) {
            const int rl = WROWS * wave + 8 * i + (lane >> 3);
            o[i] = (int64_t)min(tn0 + rl, g.N - 1) * g.ldw + lchunk(rl) * 8;
        }
    };
    auto set_offA = [&](int tm0) { a_offsets(tm0, offA); };
    auto set_offW = [&](int tn0) { w_offsets(tn0, offW); };
    // the ring switches A's and W's offsets to the next tile one K-tile apart
    auto tile_origin = [&](int tile, int& tm0, int& tn0) {
        int tm, tn;
        map_tile<TILE_GM>(tile, nblocks, tiles_m, tiles_n, tm, tn);
        tm0 = tm * DM;
        tn0 = tn * S::TBN;
    };
    auto setup_tile = [&](int tile) {
        int tm, tn;
        map_tile<TILE_GM>(tile, nblocks, tiles_m, tiles_n, tm, tn);
        m0 = tm * DM;
        n0 = tn * S::TBN;
        if constexpr (EPI == EPI_PLAIN || GROUP_EPI) skew = ((tm & 7) + 2 * tn) % nk;
        set_offA(m0);
        set_offW(n0);
    };
    // load j of A rows AROWS w + 8 j.. / of W rows WROWS w + 8 j.. at K offset k0 into stage st
    // (nx: from the next tile, ring only; a uniform select, no branch inside the MFMA sequence)
    auto issue_a = [&](int k0, bf16_t* st, int j, bool nx = false) {
        int64_t o = offA[j];
        if constexpr (RING) o = nx ? offAn[j] : o;
        __builtin_amdgcn_global_load_lds((gbl_void*)(A + o + k0), (lds_void*)(st + (AROWS * wave + 8 * j) * BK), 16, 0, 0);
    };
    auto issue_w = [&](int k0, bf16_t* st, int j, bool nx = false) {
        int64_t o = offW[j];
        if constexpr (RING) o = nx ? offWn[j] : o;
        __builtin_amdgcn_global_load_lds((gbl_void*)(W + o + k0), (lds_void*)(st + (WROWS * wave + 8 * j) * BK), 16, 0, 0);
    };
    // load j of K-tile G (both operands at k0): j < NA fills A, otherwise W
    auto issue_one = [&](int k0, int G, int j) {
        if (j < NA) issue_a(k0, a_stage(G), j);
        else issue_w(k0, w_stage(G), j - NA);
    };
    constexpr int NL = NA + NWL;                       // load instructions per wave per stage
    constexpr int LD_STEPS = 3;                        // K steps over which they are spread
    constexpr int LPS = (NL + LD_STEPS - 1) / LD_STEPS;

    f32x16 acc[NB][MB];

    // fragment rows of this lane: row0 + lane % 32 with row0 a multiple of 32, so
    // (row >> 1) & 7 == (lane >> 1) & 7
    const int frow = lane & 31, fsw = (lane >> 1) & 7, fhalf = lane >> 5;
    auto frag = [&](const bf16_t* tile, int row0, int kk) -> bf16x8 {
        const int slot = (2 * kk + fhalf) ^ fsw;
        return *(const bf16x8*)&tile[(row0 + frow) * BK + slot * 8];
    };

    // K-tile G; with_loads: also fetch, from the tiles offA/offW describe, K-tile G + 1 of both
    // operands at K offset k0a (two stages) or W's K-tile G + 1 at k0w and A's K-tile G + 2 at k0a
    // (ring); without, the load issue stays free of branches inside the MFMA sequence
    auto ktile = [&](const int G, const int k0a, const int k0w, auto with_loads, bool a_nx = false,
                     bool w_nx = false, bool has_a1 = false, bool has_a2 = false, bool has_w1 = false) {
        constexpr bool more = decltype(with_loads)::value;
        if constexpr (RING) {
            // this lane's loads of K-tile G landed: only A's K-tile G + 1 (has_a1), issued after
            // them, may still be in flight; then everyone's, and everyone left K-tile G - 1.  The
            // barrier is a bare s_barrier with a memory clobber: __syncthreads would also wait for
            // A's G + 1
            if (has_a1) __builtin_amdgcn_s_waitcnt(0x3F70 | NA);
            else __builtin_amdgcn_s_waitcnt(0x3F70);
            asm volatile("s_barrier" ::: "memory");
        } else {
            __builtin_amdgcn_s_waitcnt(0x3F70);  // vmcnt(0): this lane's loads of K-tile G landed
            __syncthreads();                      // ... everyone's; and everyone left K-tile G - 1
        }
        const bf16_t* sA = a_stage(G) + (wm * S::WM) * BK;
        const bf16_t* sW = w_stage(G) + (wn * S::WN) * BK;
        bf16x8 af[2][MB], wf[2][NB];
#pragma unroll
        for (int i = 0; i < MB; ++i) af[0][i] = frag(sA, 32 * i, 0);
#pragma unroll
        for (int i = 0; i < NB; ++i) wf[0][i] = frag(sW, 32 * i, 0);
        __builtin_amdgcn_s_waitcnt(0xC07F);       // lgkmcnt(0): the first step's fragments
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int kk = 0; kk < BK / 16; ++kk) {
            const int cur = kk & 1;
            // issue slot i: MFMAs 2i and 2i+1, fragment reads 2i-2 and 2i-1 of the next step and
            // load i of the next K-tile, fenced so the scheduler keeps the slots in order.  The reads
            // go out early in the step (after its first MFMAs) and are waited for at its end, so no
            // MFMA waits on a read of its own step.
            constexpr int NPAIR = NB * MB / 2, NREAD = MB + NB;
            // enough slots for every MFMA pair, every load and every read (two per slot from slot 1)
            constexpr int NRSLOT = (NREAD + 1) / 2 + 1;
            constexpr int NSLOT0 = NPAIR > LPS ? NPAIR : LPS;
            constexpr int NSLOT = NSLOT0 > NRSLOT ? NSLOT0 : NRSLOT;
            static_assert(2 * (NSLOT - 1) >= NREAD && NSLOT >= NPAIR && LD_STEPS * LPS >= NL &&
                          LD_STEPS < BK / 16 + 1, "every read, MFMA pair and load has a slot");
            const int nload = (more && kk < LD_STEPS) ? min(LPS, NL - kk * LPS) : 0;
#pragma unroll
            for (int i = 0; i < NSLOT; ++i) {
                if (i < NPAIR) {
                    // 256-wide tiles: the wave issuing an MFMA pair wins the SIMD's arbitration
                    // over its partner (MLP up 86.4-87.0 -> 85.4-85.5 us, vocabulary projection -2.5 %
                    // at B16 L1024; on the 192-wide tiles the same made MLP down 4 % slower)
                    if constexpr (S::TBN == 256) __builtin_amdgcn_s_setprio(1);
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const int q = 2 * i + h, nb = q / MB, mb = q % MB;
                        acc[nb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[cur][nb], af[cur][mb], acc[nb][mb], 0, 0, 0);
                    }
                    if constexpr (S::TBN == 256) __builtin_amdgcn_s_setprio(0);
                }
                if (kk + 1 < BK / 16 && i >= 1) {
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const int r = 2 * (i - 1) + h;
                        if (r < MB) af[cur ^ 1][r] = frag(sA, 32 * r, kk + 1);
                        else if (r < NREAD) wf[cur ^ 1][r - MB] = frag(sW, 32 * (r - MB), kk + 1);
                    }
                }
                if constexpr (more)
                    if (i < nload) {
                        const int j = kk * LPS + i;
                        if constexpr (RING) {
                            // W first: see the wait above; past the last tile nothing is fetched
                            if (j < NWL) {
                                if (has_w1) issue_w(k0w, w_stage(G + 1), j, w_nx);
                            } else if (has_a2) {
                                issue_a(k0a, a_stage(G + 2), j - NWL, a_nx);
                            }
                        } else {
                            issue_one(k0a, G + 1, j);
                        }
                    }
                __builtin_amdgcn_sched_barrier(0);
            }
            if (kk + 1 < BK / 16) __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // bias of this lane's output columns (4 consecutive per (nb, j4)); the bf16-output epilogues
    // fetch it ahead of the K loop, the residual epilogue (short of registers) when it needs it
    auto load_bias4 = [&](int nb, int j4) -> uint2 {
        const int n = n0 + wn * S::WN + nb * 32 + 8 * j4 + 4 * (lane >> 5);
        const bf16_t* bp = (const bf16_t*)g.bias + n;
        if (n + 3 < g.N) return *(const uint2*)bp;
        uint32_t h[4] = {0u, 0u, 0u, 0u};
        for (int e = 0; e < 4; ++e)
            if (n + e < g.N) h[e] = bp[e];
        return make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
    };
    constexpr bool PREFETCH_BIAS = EPI == EPI_BIAS || EPI == EPI_BIAS_GELU;
    uint2 braw[PREFETCH_BIAS ? NB : 1][4];
    auto prefetch_bias = [&]() {
        if constexpr (PREFETCH_BIAS) {
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int j4 = 0; j4 < 4; ++j4) braw[nb][j4] = load_bias4(nb, j4);
        }
    };
    auto bias4 = [&](int nb, int j4, float* b4) {
        uint2 r = make_uint2(0u, 0u);
        if constexpr (PREFETCH_BIAS) r = braw[nb][j4];
        else if constexpr (EPI != EPI_PLAIN && EPI != EPI_GATE && !GROUP_EPI) r = load_bias4(nb, j4);
        b4[0] = bf16_lo(r.x); b4[1] = bf16_hi(r.x); b4[2] = bf16_lo(r.y); b4[3] = bf16_hi(r.y);
    };

    // epilogue of the tile at (m0, n0); n0 and the bias are read through the lambdas above, so the
    // caller keeps them describing this tile until the epilogue is done
    auto epilogue = [&](const int tm0, const int Gl) {
        if constexpr (EPI == EPI_BIAS_RESID) {
            // The accumulators started from the residual h (loaded with the tile's first K-tile),
            // so the epilogue only stores h + A W^T + bias.  One 32 x 32 block at a time goes
            // through this wave's 4 KB of LDS (above stage 0) so that eight lanes write one 128-byte
            // row segment (an MFMA lane holds four columns of 32 different rows).  Chunk slots are
            // XOR-swizzled by row like the operand tiles (slot = chunk ^ ((row >> 1) & 7)), which
            // keeps the row-per-lane writes and the row-segment reads free of bank conflicts.
            __syncthreads();                      // every wave is done with the operand stages
            // staging above stage 0 (two stages: the next tile's first K-tile streams into stage 0), or
            // in the A stage of the last K-tile (ring: the next tile's loads go to the other stages)
            float* cst = (RING ? (float*)a_stage(Gl) : (float*)(smem + S::STAGE)) + wave * (32 * 32);
            float* C = (float*)g.C;
            const bf16_t* bias = (const bf16_t*)g.bias;
            const int rr = lane >> 3, c4 = (lane & 7) * 4;    // read-back: row rr + 8 it, columns c4..
#pragma unroll
            for (int b = 0; b < MB * NB; ++b) {
                const int mb = b % MB, nb = b / MB;
                const int wr = lane & 31;
#pragma unroll
                for (int j4 = 0; j4 < 4; ++j4) {
                    const int slot = (2 * j4 + (lane >> 5)) ^ ((wr >> 1) & 7);
                    *(float4*)&cst[wr * 32 + slot * 4] =
                        make_float4(acc[nb][mb][4 * j4], acc[nb][mb][4 * j4 + 1], acc[nb][mb][4 * j4 + 2],
                                    acc[nb][mb][4 * j4 + 3]);
                }
                const int n = n0 + wn * S::WN + nb * 32 + c4;
                float bv[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (n + e < g.N) bv[e] = bf16_to_f32(bias[n + e]);
#pragma unroll
                for (int it = 0; it < 4; ++it) {
                    const int r = rr + 8 * it;
                    const float4 v = *(const float4*)&cst[r * 32 + (((c4 >> 2) ^ ((r >> 1) & 7)) * 4)];
                    const int m = tm0 + wm * S::WM + mb * 32 + r;
                    if (m >= M) continue;
                    float* dst = C + (int64_t)m * g.ldc + n;
                    if (n + 3 < g.N) {
                        // an ordinary store: the normalisation reads the row next and finds it in
                        // the Infinity Cache (12.9 -> 11.9 us per LayerNorm at B16 L1024)
                        *(f32x4*)dst = f32x4{v.x + bv[0], v.y + bv[1], v.z + bv[2], v.w + bv[3]};
                    } else {
                        const float o[4] = {v.x + bv[0], v.y + bv[1], v.z + bv[2], v.w + bv[3]};
                        for (int e = 0; e < 4; ++e)
                            if (n + e < g.N) dst[e] = o[e];
                    }
                }
            }
        } else {
            // bf16 outputs: each wave stages half of its WM x WN sub-tile at a time in LDS (rows
            // padded by 16 B, above stage 0), then writes whole row segments with 16-byte stores.
            __syncthreads();                      // every wave is done with the operand stages
            bf16_t* cst = smem + S::STAGE + wave * (S::WM / 2 * S::CSTR);
            bf16_t* C = (bf16_t*)g.C;
            const int mrow0 = tm0 + wm * S::WM, ncol0 = n0 + wn * S::WN;
            // e.g. WN = 64: 8 chunks per row, 8 rows per wave instruction; WN = 96: 12 chunks per
            // row, 5 rows per instruction (lanes 60..63 idle)
            constexpr int CPR = S::WN / 8;            // 16-byte chunks per staged row
            constexpr int RPI = 64 / CPR;             // rows per wave instruction
            float rs[EPI == EPI_GATE ? MB : 1];       // gate factor of this lane's rows
            if constexpr (EPI == EPI_GATE) {
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) rs[mb] = gate_row_scale(g, mrow0 + mb * 32 + (lane & 31));
            }
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                if constexpr (EPI == EPI_LSE_CDF) break;   // the store-free draw keeps no logits
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                    for (int j4 = 0; j4 < 4; ++j4) {
                        const int nl = nb * 32 + 8 * j4 + 4 * (lane >> 5);
                        float b4[4];
                        bias4(nb, j4, b4);
#pragma unroll
                        for (int mh = 0; mh < MB / 2; ++mh) {
                            const int mb = half * (MB / 2) + mh;
                            float o[4];
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                float x = acc[nb][mb][4 * j4 + e] + b4[e];
                                if (EPI == EPI_BIAS_GELU) x = gelu_tanh(x);
                                if constexpr (EPI == EPI_GATE) x = acc[nb][mb][4 * j4 + e] * rs[mb];
                                o[e] = x;
                            }
                            uint2 pk;
                            pk.x = pack_bf16x2(o[0], o[1]);
                            pk.y = pack_bf16x2(o[2], o[3]);
                            *(uint2*)&cst[(mh * 32 + (lane & 31)) * S::CSTR + nl] = pk;
                        }
                    }
                for (int r0 = 0; r0 < S::WM / 2; r0 += RPI) {
                    const int r = r0 + lane / CPR, c = (lane % CPR) * 8;
                    if (lane >= RPI * CPR || r >= S::WM / 2) continue;
                    const int m = mrow0 + half * (S::WM / 2) + r, n = ncol0 + c;
                    if (m >= M || n >= g.N) continue;
                    const uint4 v = *(const uint4*)&cst[r * S::CSTR + c];
                    bf16_t* dst = C + (int64_t)m * g.ldc + n;
                    if (n + 7 < g.N) {
                        // the QKV output is stored normally: the attention reads it next, from the
                        // Infinity Cache (attention 66.8-69.5 -> 63.5-67.4 us, QKV +0.4-0.9 us)
                        if constexpr (EPI == EPI_BIAS) *(u32x4*)dst = u32x4{v.x, v.y, v.z, v.w};
                        else __builtin_nontemporal_store(u32x4{v.x, v.y, v.z, v.w}, (u32x4*)dst);
                    } else {
                        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
                        for (int e = 0; n + e < g.N; ++e) dst[e] = (bf16_t)((w[e >> 1] >> (16 * (e & 1))) & 0xFFFFu);
                    }
                }
            }
            if constexpr (GROUP_EPI) {
                // Log-sum-exp of each tile row over the tile's 256 columns (one sampling group), taken
                // over the rounded values just stored.  Rounding is monotonic, so the row maximum is
                // the rounded maximum of the accumulators.  A wave covers 64 columns of a row (lanes
                // l and l ^ 32 hold 32 each); the WGN partial (max, sum) pairs of a row meet in LDS
                // past the staging area.  Columns past N (clamped W rows) do not count.
                static_assert(S::TBN == DD_GUMBEL_GROUP, "one tile column = one sampling group");
                float2* part = (float2*)((char*)smem + S::LDS);
                const int nl0 = ncol0 + 4 * (lane >> 5);
                // store-free draw: the chunk sums of every tile row, [DM][CHK_LD] floats with chunk
                // c of row r at slot c ^ (r & 31), so that 32 rows written (or scanned) at once hit
                // 32 banks, in operand stage 1: the last K-tile read it and the next tile's first
                // K-tile loads go to stage 0
                constexpr int CHK_LD = S::TBN / 4;
                static_assert(EPI != EPI_LSE_CDF || (CHK_LD == 64 && (size_t)S::DM * CHK_LD * sizeof(float) <=
                                                                      S::STAGE * sizeof(bf16_t)),
                              "chunk sums fit in one operand stage");
                float* chk = (float*)(smem + S::STAGE);
                auto rows_partial = [&](auto ragged_c) {
                    constexpr bool ragged = decltype(ragged_c)::value;
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb) {
                        float mx = -INFINITY;
#pragma unroll
                        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                            for (int j4 = 0; j4 < 4; ++j4)
#pragma unroll
                                for (int e = 0; e < 4; ++e)
                                    if (!ragged || nl0 + nb * 32 + 8 * j4 + e < g.N)
                                        mx = fmaxf(mx, acc[nb][mb][4 * j4 + e]);
                        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
                        const float mr = bf16_to_f32(f32_to_bf16(mx));
                        const float moff = (mr == -INFINITY ? 0.f : mr) * -LOG2E_F;
                        // sums over chunks of 4 consecutive classes first (lanes l and l ^ 32 hold
                        // alternate chunks); the store-free draw keeps them in LDS for its scan
                        float sum = 0.f;
#pragma unroll
                        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                            for (int j4 = 0; j4 < 4; ++j4) {
                                float cs = 0.f;
#pragma unroll
                                for (int e = 0; e < 4; ++e) {
                                    float v = round_bf16(acc[nb][mb][4 * j4 + e]);
                                    if (ragged && nl0 + nb * 32 + 8 * j4 + e >= g.N) v = -INFINITY;
                                    cs += __builtin_amdgcn_exp2f(fmaf(v, LOG2E_F, moff));
                                }
                                if constexpr (EPI == EPI_LSE_CDF)
                                    chk[(wm * S::WM + mb * 32 + (lane & 31)) * CHK_LD +
                                        ((wn * 16 + nb * 8 + 2 * j4 + (lane >> 5)) ^ (lane & 31))] = cs;
                                sum += cs;
                            }
                        sum += __shfl_xor(sum, 32, 64);
                        if (lane < 32) part[(wm * S::WM + mb * 32 + lane) * S::WGN + wn] = make_float2(mr, sum);
                    }
                };
                if (n0 + S::TBN <= g.N) rows_partial(std::false_type{});
                else rows_partial(std::true_type{});
                __syncthreads();
                // store-free draw: per tile row, the wave whose 64 columns hold the crossing of the
                // running sum and the remaining target in that wave's own reference (wave -1: none)
                float2* sel = part + DM * S::WGN;
                const int grp = n0 / DD_GUMBEL_GROUP;
                if (tid < DM && tm0 + tid < M) {
                    float2 p[S::WGN];
                    float mm = -INFINITY;
#pragma unroll
                    for (int w = 0; w < S::WGN; ++w) {
                        p[w] = part[tid * S::WGN + w];
                        mm = fmaxf(mm, p[w].x);
                    }
                    const float mref = mm == -INFINITY ? 0.f : mm;
                    float sum = 0.f;
#pragma unroll
                    for (int w = 0; w < S::WGN; ++w) sum += p[w].y * exp2f((p[w].x - mref) * LOG2E_F);
                    g.lse[(int64_t)(tm0 + tid) * g.lse_ld + grp] = mref + logf(sum);
                    if constexpr (EPI == EPI_LSE_CDF) {
                        // the row's target t = u S; the wave sums (scaled to the common reference)
                        // in class order give the crossing wave, a scan of that wave's 16 chunk
                        // sums the crossing chunk and the remaining target in the wave's reference
                        const int m = tm0 + tid;
                        const uint32_t grow = g.row0 + (uint32_t)(g.row_ids ? g.row_ids[m] : g.a_rows ? g.a_rows[m] : m);
                        const uint32_t word = counter_word(g.seed, STREAM_GROUP_U, g.step, grow, (uint32_t)grp);
                        const float t = (float)(((double)word + 0.5) * 0x1p-32 * (double)sum);
                        const float* crow = chk + tid * CHK_LD;
                        // the crossing wave from the wave sums, then its 16 chunks
                        float cum = 0.f, tw = 0.f;
                        int wsel = -1, wlast = -1;
#pragma unroll
                        for (int w = 0; w < S::WGN; ++w) {
                            const float add = p[w].y * exp2f((p[w].x - mref) * LOG2E_F);
                            if (add > 0.f) wlast = w;
                            if (wsel < 0 && cum + add > t) {
                                wsel = w;
                                tw = (t - cum) / exp2f((p[w].x - mref) * LOG2E_F);
                            }
                            cum += add;
                        }
                        if (wsel < 0) {          // rounding left no crossing: the last wave with mass
                            wsel = wlast;
                            tw = INFINITY;
                        }
                        float tres = 0.f;
                        int csel = -1, clast = -1;
                        if (wsel >= 0) {
                            float cc = 0.f;
#pragma unroll 4
                            for (int c = 0; c < 16; ++c) {
                                const float cw = crow[(wsel * 16 + c) ^ (tid & 31)];
                                if (cw > 0.f) clast = wsel * 16 + c;
                                if (csel < 0 && cc + cw > tw) {
                                    csel = wsel * 16 + c;
                                    tres = tw - cc;
                                }
                                cc += cw;
                            }
                            if (csel < 0) {      // the wave's scan fell short of its sum: its last chunk
                                csel = clast;
                                tres = INFINITY;
                            }
                        }
                        sel[tid] = make_float2(tres, __int_as_float(csel));
                        if (csel < 0) g.cand[(int64_t)m * g.cand_ld + grp] = -1;   // no finite logit
                    }
                }
                if constexpr (EPI == EPI_LSE_CDF) {
                    // the lane holding the crossing chunk of a row scans its 4 classes, from its
                    // accumulators and its wave's row maximum
                    __syncthreads();
                    const int myh = lane >> 5;
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb) {
                        const int rl = wm * S::WM + mb * 32 + (lane & 31);
                        const float2 sl = sel[rl];
                        const int c = __float_as_int(sl.y);
                        if (tm0 + rl >= M || c < 0 || (c >> 4) != wn || (c & 1) != myh) continue;
                        const int q = (c & 15) >> 1;      // nb * 4 + j4
                        float a4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                            for (int j4 = 0; j4 < 4; ++j4)
#pragma unroll
                                for (int e = 0; e < 4; ++e)
                                    a4[e] = (nb * 4 + j4 == q) ? acc[nb][mb][4 * j4 + e] : a4[e];
                        const float mr = part[rl * S::WGN + wn].x;
                        const float moff = (mr == -INFINITY ? 0.f : mr) * -LOG2E_F;
                        const int n0c = nl0 + 32 * (q >> 2) + 8 * (q & 3);   // class of a4[0]
                        int ce = -1, le = -1;
                        float c2 = 0.f;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const float v = n0c + e < g.N ? round_bf16(a4[e]) : -INFINITY;
                            const float x = __builtin_amdgcn_exp2f(fmaf(v, LOG2E_F, moff));
                            if (x > 0.f) le = e;
                            if (ce < 0 && c2 + x > sl.x) ce = e;
                            c2 += x;
                        }
                        if (ce < 0) ce = le;
                        g.cand[(int64_t)(tm0 + rl) * g.cand_ld + grp] = ce < 0 ? -1 : n0c + ce;
                    }
                }
            }
        }
    };

    setup_tile(L);
    prefetch_bias();
    if constexpr (RING) {
        // W's K-tile 0, then A's K-tiles 0 and 1 (nk >= 2)
#pragma unroll
        for (int j = 0; j < NWL; ++j) issue_w(0, w_stage(0), j);
#pragma unroll
        for (int j = 0; j < NA; ++j) issue_a(0, a_stage(0), j);
#pragma unroll
        for (int j = 0; j < NA; ++j) issue_a(BK, a_stage(1), j);
    } else {
#pragma unroll
        for (int j = 0; j < NL; ++j) issue_one(skew * BK, 0, j);
    }
    int G = 0;                                    // K-tiles begun by this workgroup
    while (true) {
        const int cskew = skew;
        if constexpr (EPI == EPI_BIAS_RESID) {
            // residual epilogue: start from h (this lane's MFMA output positions), fetched together
            // with the tile's first K-tile instead of after the K loop.  h is C itself, or (not in
            // the ring form) the rows of c_in that c_rows lists
            const float* C = (const float*)g.C;
            int64_t hrow[MB];
#pragma unroll
            for (int j = 0; j < MB; ++j) {
                const int m = m0 + wm * S::WM + j * 32 + (lane & 31);
                hrow[j] = m;
                if constexpr (!RING) {
                    if (g.c_in && g.c_rows && m < M) hrow[j] = g.c_rows[m];
                }
            }
            if constexpr (!RING) {
                if (g.c_in) C = g.c_in;
            }
#pragma unroll
            for (int i = 0; i < NB; ++i)
#pragma unroll
                for (int j = 0; j < MB; ++j)
#pragma unroll
                    for (int j4 = 0; j4 < 4; ++j4) {
                        const int m = m0 + wm * S::WM + j * 32 + (lane & 31);
                        const int n = n0 + wn * S::WN + i * 32 + 8 * j4 + 4 * (lane >> 5);
                        float4 h = make_float4(0.f, 0.f, 0.f, 0.f);
                        if (m < M && n + 3 < g.N) {
                            h = *(const float4*)(C + hrow[j] * g.ldc + n);
                        } else if (m < M) {
                            float t[4] = {0.f, 0.f, 0.f, 0.f};
                            for (int e = 0; e < 4; ++e)
                                if (n + e < g.N) t[e] = C[hrow[j] * g.ldc + n + e];
                            h = make_float4(t[0], t[1], t[2], t[3]);
                        }
                        acc[i][j][4 * j4] = h.x;
                        acc[i][j][4 * j4 + 1] = h.y;
                        acc[i][j][4 * j4 + 2] = h.z;
                        acc[i][j][4 * j4 + 3] = h.w;
                    }
        } else {
#pragma unroll
            for (int i = 0; i < NB; ++i)
#pragma unroll
                for (int j = 0; j < MB; ++j)
#pragma unroll
                    for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
        }
        const int Ln = L + (int)gridDim.x;
        const bool next = Ln < nblocks;
        const int tm0 = m0;
        if constexpr (RING) {
            int tm_n = m0, tn_n = n0;
            if (next) tile_origin(Ln, tm_n, tn_n);
            a_offsets(tm_n, offAn);
            w_offsets(tn_n, offWn);
        }
        for (int t = 0; t < nk; ++t, ++G) {
            if constexpr (RING) {
                // A's loads move to the next tile one K-tile before W's: K-tile nk - 2 fetches A's
                // first K-tile of the next tile, K-tile nk - 1 W's first and A's second (uniform
                // branches around the loads; after the last tile nothing is fetched, so the
                // epilogue's barrier has no load to wait for)
                const int k0w = t + 1 < nk ? (t + 1) * BK : 0;
                const int k0a = t + 2 < nk ? (t + 2) * BK : (t + 2 - nk) * BK;
                ktile(G, k0a, k0w, std::true_type{}, t + 2 >= nk, t + 1 >= nk, t + 1 < nk || next,
                      t + 2 < nk || next, t + 1 < nk || next);
            } else {
                if (t == nk - 1 && next) {        // the last K-tile fetches the next tile's first one
                    const int tn0 = n0;
                    setup_tile(Ln);
                    n0 = tn0;                     // the epilogue still describes this tile
                }
                // the last K-tile fetches the next tile's first K-slice (after the very last tile it
                // re-fetches slice 0 into stage 0: unused, in bounds; one call site keeps the MFMA
                // sequence in one copy)
                const int next_k0 = t + 1 < nk ? ((t + 1 + cskew) % nk) * BK : (next ? skew * BK : 0);
                ktile(G, next_k0, 0, std::true_type{});
            }
        }
        if constexpr (RING) {
#pragma unroll
            for (int i = 0; i < NA; ++i) offA[i] = offAn[i];
#pragma unroll
            for (int i = 0; i < NWL; ++i) offW[i] = offWn[i];
        }
        epilogue(tm0, G - 1);
        if (!next) break;
        int tm_n, tn_n;
        map_tile<TILE_GM>(Ln, nblocks, tiles_m, tiles_n, tm_n, tn_n);
        m0 = tm_n * DM;
        n0 = tn_n * S::TBN;
        prefetch_bias();
        L = Ln;
    }
    __builtin_amdgcn_s_waitcnt(0x3F70);           // vmcnt(0): no LDS write in flight at exit
}

template <int TBM, int TBN>
constexpr size_t gemm_lds_bytes() { return (size_t)2 * (TBM + TBN) * LSTR * sizeof(bf16_t); }

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
            if (EPI == EPI_GATE) x *= gate_row_scale(g, m);
            else if (EPI != EPI_PLAIN) x += ((const float*)g.bias)[n];
            if (EPI == EPI_BIAS_GELU) x = 0.5f * x * (1.0f + tanhf(0.7978845608028654f * (x + 0.044715f * x * x * x)));
            float* c = (float*)g.C + (int64_t)m * g.ldc + n;
            if (EPI == EPI_BIAS_RESID) *c += x;
            else *c = x;
        }
    }
}

template <int TBM, int TBN, int EPI>
static void launch_tile(const GemmArgs& g, hipStream_t s) {
    const int tm = (g.M + TBM - 1) / TBM, tn = (g.N + TBN - 1) / TBN;
    constexpr size_t lds = gemm_lds_bytes<TBM, TBN>();
    static bool attr = false;   // one-time opt-in to more than 64 KB of LDS per workgroup
    if (!attr) {
        (void)hipFuncSetAttribute((const void*)gemm_bf16_kernel<TBM, TBN, EPI>,
                                  hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        attr = true;
    }
    launch_k((gemm_bf16_kernel<TBM, TBN, EPI>), dim3(tm * tn), dim3(256), lds, s, g, tm, tn);
}

// Tile choice for the direct-to-LDS kernel: the N width (256 or 192) with the smaller estimated time,
// counting whole rounds of workgroups over the CUs (a round of 192-wide tiles takes about 0.85 of a
// round of 256-wide ones on MI355X), in the 8-wavefront form (two wavefronts per SIMD, measured 2-6%
// faster than four wavefronts of twice the sub-tile).  K % 128 != 0 falls back to the 128 x 128
// register-staged kernel.  Skinny products (N <= 128, e.g. an adapter down-projection to rank r)
// would leave most CUs idle with 256-row tiles (M / 256 workgroups): with K % 128 == 0 they take
// 64 x 32 direct-to-LDS tiles of one wavefront, up to eight workgroups per CU (their K loop is
// latency-bound, so more independent loops per CU pay: 12 % faster than one 64 x 128 workgroup of
// four wavefronts per CU), else 64 x 128 register-staged tiles.  DD_GEMM_TILE (0..10) forces a
// variant for tuning and tests (4: 256 x 256 / 4 waves, 5: 256 x 192 / 4 waves, 6: 256 x 256 /
// 8 waves, 7: 256 x 192 / 8 waves, 8: 64 x 128 register-staged, 9: 64 x 128 direct-to-LDS,
// 10: 64 x 32 direct-to-LDS / 1 wave).
static int num_cus() {
    static int n = 0;
    if (n == 0) {
        int dev = 0, v = 0;
        (void)hipGetDevice(&dev);
        n = (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0) ? v : 256;
    }
    return n;
}

static int pick_tile(const GemmArgs& g) {
    const char* e = getenv("DD_GEMM_TILE");
    const int forced = e ? atoi(e) : -1;
    if (((forced >= 4 && forced <= 7) || forced >= 9) && g.K % (2 * BK) != 0) return 0;
    const bool gathered = g.a_rows || g.m_count || g.c_in;   // only the direct-to-LDS kernels
    if (forced >= 0 && forced <= 10 && !(gathered && (forced < 4 || forced == 8))) return forced;
    if (g.N <= 128) return g.K % (2 * BK) == 0 ? 10 : (gathered ? 0 : 8);
    if (g.K % (2 * BK) != 0) return 0;
    const int64_t ncu = num_cus();
    const int64_t tm = (g.M + DM - 1) / DM;
    const int64_t r256 = (tm * ((g.N + 255) / 256) + ncu - 1) / ncu;
    const int64_t r192 = (tm * ((g.N + 191) / 192) + ncu - 1) / ncu;
    return (17 * r192 < 20 * r256) ? 7 : 6;
}

template <int EPI, int ROLE, int TBN, int WGM, int WGN, int DMR = DM>
static void launch_dl(const GemmArgs& g, hipStream_t s) {
    using S = DLShape<TBN, WGM, WGN, DMR>;
    constexpr size_t lds = dl_lds_bytes<EPI, S>();
    static_assert(lds <= 160 * 1024, "LDS");
    const int tm = (g.M + S::DM - 1) / S::DM, tn = (g.N + S::TBN - 1) / S::TBN;
    static bool attr = false;
    if (!attr) {
        (void)hipFuncSetAttribute((const void*)gemm_bf16_dl_kernel<EPI, ROLE, TBN, WGM, WGN, DMR>,
                                  hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        attr = true;
    }
    // persistent: at most WG_PER_CU workgroups per CU
    const int grid = (int)std::min<int64_t>((int64_t)tm * tn, (int64_t)num_cus() * S::WG_PER_CU);
    launch_k((gemm_bf16_dl_kernel<EPI, ROLE, TBN, WGM, WGN, DMR>), dim3(grid), dim3(S::THREADS), lds,
                       s, g, tm, tn);
}

template <int EPI, int ROLE>
static void launch_epi(int dtype, const GemmArgs& g, hipStream_t s) {
    if (dtype == DD_BF16) {
        int tile = g.tile_hint > 0 ? g.tile_hint - 1 : pick_tile(g);
        // the ring instance of the 256 x 192 tile takes no gathered rows and no separate residual
        // input: the four-wavefront form
        if (tile == 7 && (g.a_rows || g.c_in) && dl_ring<EPI, DLShape<192, 4, 2>>()) tile = 5;
        switch (tile) {
            case 7: launch_dl<EPI, ROLE, 192, 4, 2>(g, s); break;
            case 6: launch_dl<EPI, ROLE, 256, 2, 4>(g, s); break;
            case 5: launch_dl<EPI, ROLE, 192, 2, 2>(g, s); break;
            case 4: launch_dl<EPI, ROLE, 256, 2, 2>(g, s); break;
            case 9: launch_dl<EPI, ROLE, 128, 1, 4, 64>(g, s); break;
            case 10: launch_dl<EPI, ROLE, 32, 1, 1, 64>(g, s); break;
            case 8: launch_tile<64, 128, EPI>(g, s); break;
            case 3: launch_tile<256, 256, EPI>(g, s); break;
            case 2: launch_tile<256, 128, EPI>(g, s); break;
            case 1: launch_tile<128, 256, EPI>(g, s); break;
            default: launch_tile<128, 128, EPI>(g, s); break;
        }
    } else {
        const int tm = (g.M + FT - 1) / FT, tn = (g.N + FT - 1) / FT;
        launch_k(gemm_f32_kernel<EPI>, dim3(tm * tn), dim3(256), 0, s, g, tm, tn);
    }
}

bool gemm_gather_supported(int dtype, int K) { return dtype == DD_BF16 && K % (2 * BK) == 0; }
bool gemm_lse_supported(int dtype, int K) { return dtype == DD_BF16 && K % (2 * BK) == 0; }

dd_status launch_gemm(int dtype, int epi, int cls, const GemmArgs& g, hipStream_t s) {
    if (g.M == 0 || g.N == 0) return DD_OK;
    if (g.K <= 0) {
        set_error("GEMM with K = %d", g.K);
        return DD_E_ARG;
    }
    if ((g.a_rows || g.m_count || g.c_in || g.c_rows || g.row_ids) && !gemm_gather_supported(dtype, g.K)) {
        set_error("row-gathered GEMM needs the bf16 path and K %% 128 == 0");
        return DD_E_UNSUPPORTED;
    }
    if (g.m_gate > 0 && !g.m_count) {
        set_error("a row-count gate needs the device-side row count");
        return DD_E_ARG;
    }
    if ((g.c_in && epi != EPI_BIAS_RESID) || (g.c_rows && !g.c_in)) {
        set_error("a separate residual input (and its row list) needs the residual epilogue");
        return DD_E_ARG;
    }
    if ((epi == EPI_LSE || epi == EPI_LSE_CDF) &&
        (!gemm_lse_supported(dtype, g.K) || !g.lse || g.lse_ld < (g.N + 255) / 256)) {
        set_error("group log-sum-exp epilogue needs the bf16 path, K %% 128 == 0 and an lse buffer");
        return DD_E_UNSUPPORTED;
    }
    if (epi == EPI_LSE_CDF && (!g.cand || g.cand_ld < (g.N + 255) / 256)) {
        set_error("store-free draw epilogue needs a candidate buffer");
        return DD_E_UNSUPPORTED;
    }
    ProfScope ps(cls, s);
    switch (epi) {
        case EPI_BIAS: launch_epi<EPI_BIAS, KC_GEMM_QKV>(dtype, g, s); break;
        case EPI_BIAS_GELU: launch_epi<EPI_BIAS_GELU, KC_GEMM_MLP1>(dtype, g, s); break;
        case EPI_BIAS_RESID:
            if (cls == KC_GEMM_O) launch_epi<EPI_BIAS_RESID, KC_GEMM_O>(dtype, g, s);
            else launch_epi<EPI_BIAS_RESID, KC_GEMM_MLP2>(dtype, g, s);
            break;
        case EPI_GATE: launch_epi<EPI_GATE, KC_GEMM_LORA>(dtype, g, s); break;
        // one tile column per sampling group: always the 256-wide, 8-wavefront tile
        case EPI_LSE: launch_dl<EPI_LSE, KC_GEMM_VOCAB, 256, 2, 4>(g, s); break;
        case EPI_LSE_CDF: launch_dl<EPI_LSE_CDF, KC_GEMM_VOCAB, 256, 2, 4>(g, s); break;
        default: launch_epi<EPI_PLAIN, KC_GEMM_VOCAB>(dtype, g, s); break;
    }
    return launch_status("gemm");
}

}  // namespace dd
