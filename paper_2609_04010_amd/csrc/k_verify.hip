// Speculative verification of drafted blocks (Alg. 1, linear sampler).
//
// For sequence s the target logits p_1..p_B and the draft logits q_1..q_{B-1} are rows of two
// [rows][ld] matrices, the drafted tokens x_1..x_{B-1} a [S][B-1] array.  With acceptance uniforms
// u_i (word (STREAM_VERIFY, step, row0 + s, i)):
//   n = first i with u_i > min(1, p_i(x_i) / q_i(x_i)), else B
//   z ~ Norm([p_n - q_n]_+) if n < B, else z ~ p_B     (p_n itself if the residual has no mass)
// Rows whose logits give no valid draw (NaN, +inf, no finite logit) set DD_DEVERR_LOGITS and
// emit z = 0.
// z is drawn with the two-level Gumbel-max of the posterior kernel (groups of DD_GUMBEL_GROUP
// classes, no mask group): the draw is invariant to the normaliser, so group masses and class
// scores use the unnormalised residual.
//
// Kernel 1 (one workgroup per logit row): row log-sum-exp in fp32.
// Kernel 2 (one workgroup per sequence): n from the B - 1 acceptance tests, then one pass over the
// chosen row pair for the group masses and the two-level draw.
#include <math.h>

#include <mutex>

#include "elem.h"
#include "kernels.h"
#include "rng.h"

namespace dd {

namespace {

constexpr int VT = 256;   // threads per workgroup

// Row r < S B is target row r; otherwise draft row r - S B.  One pass over the row: each thread keeps
// a running maximum m and the sum of exp(l - m), rescaled when m rises; the workgroup then combines
// the (m, sum) pairs.  The result is that of the two-pass definition: NaN if a logit is NaN, else
// +inf if one is +inf, else -inf if none is finite.
// The pass is bound by VALU work per logit, so the hot loop spends four full-rate operations and one
// exp2 per logit: a thread takes VU chunks at a time (loaded together, the next VU loaded while these
// are reduced), takes their maximum with fmax (which passes over NaN), rescales its sum when the
// maximum rises, and adds exp2(l log2 e - m log2 e).  A NaN or +inf logit makes that sum NaN
// (exp2 of NaN, or of inf - inf), so such rows are told apart afterwards by a second scan that
// only they take.
constexpr int VU = 4;
template <typename T>
__global__ __launch_bounds__(VT) void row_lse_kernel(VerifyArgs a, float* lse) {
    __shared__ float sh_m[VT / 64], sh_s[VT / 64];
    __shared__ int sh_f[VT / 64];
    constexpr int E = Elem<T>::E;
    const int r = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int np = a.S * a.B;
    const char* rowp = r < np ? (const char*)a.p + (size_t)r * a.ld * sizeof(T)
                              : (const char*)a.q + (size_t)(r - np) * a.ld * sizeof(T);
    const int V = a.V, nchunk = (V + E - 1) / E;
    float m = -INFINITY, sum = 0.f;
    constexpr int TS = VU * VT;   // chunks per tile
    // chunks c0 + u VT + tid, u < VU; chunks past the row read as -inf, and so does the part of the
    // last chunk past V
    auto load = [&](uint4 (&x)[VU], int c0) {
#pragma unroll
        for (int u = 0; u < VU; ++u) {
            const int c = c0 + u * VT + tid;
            x[u] = c < nchunk ? *(const uint4*)(rowp + (size_t)c * 16) : Elem<T>::NEG_INF4;
            if (V % E != 0 && c == nchunk - 1) Elem<T>::clip(x[u], V % E);
        }
    };
    auto absorb = [&](const uint4 (&x)[VU]) {
        float cm = -INFINITY;
#pragma unroll
        for (int u = 0; u < VU; ++u)
#pragma unroll
            for (int e = 0; e < E; ++e) cm = fmaxf(cm, Elem<T>::get(x[u], e));
        if (cm > m) {
            sum *= __builtin_amdgcn_exp2f((m - cm) * LOG2E);   // m = -inf: sum is 0 already
            m = cm;
        }
        const float moff = m == -INFINITY ? 0.f : -m * LOG2E;
#pragma unroll
        for (int u = 0; u < VU; ++u)
#pragma unroll
            for (int e = 0; e < E; ++e) sum += __builtin_amdgcn_exp2f(fmaf(Elem<T>::get(x[u], e), LOG2E, moff));
    };
    uint4 xa[VU], xb[VU];
    load(xa, 0);
    for (int c0 = 0; c0 < nchunk; c0 += 2 * TS) {
        const bool more = c0 + TS < nchunk;
        if (more) load(xb, c0 + TS);
        absorb(xa);
        if (!more) break;
        if (c0 + 2 * TS < nchunk) load(xa, c0 + 2 * TS);
        absorb(xb);
    }
    // workgroup: maximum, then the sums rescaled to it
    float M = wave_max(m);
    if (lane == 0) sh_m[wave] = M;
    __syncthreads();
    M = sh_m[0];
#pragma unroll
    for (int w = 1; w < VT / 64; ++w) M = fmaxf(M, sh_m[w]);
    const float Mref = M == -INFINITY ? 0.f : M;
    // a thread that met no finite logit has sum 0, or NaN if it met a NaN: kept as it is
    float part = m == -INFINITY ? sum : sum * __builtin_amdgcn_exp2f((m - Mref) * LOG2E);
    part = wave_sum(part);
    if (lane == 0) sh_s[wave] = part;
    __syncthreads();
    float S = sh_s[0];
#pragma unroll
    for (int w = 1; w < VT / 64; ++w) S += sh_s[w];
    if (!(S == S) || M == INFINITY) {
        // a NaN or +inf logit (the sum is NaN): NaN if any logit is NaN, else +inf
        int fl = 0;
        for (int c = tid; c < nchunk; c += VT) {
            uint4 x = *(const uint4*)(rowp + (size_t)c * 16);
            if (V % E != 0 && c == nchunk - 1) Elem<T>::clip(x, V % E);
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const float t = Elem<T>::get(x, e);
                fl |= (t != t) ? 1 : (t == INFINITY ? 2 : 0);
            }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) fl |= __shfl_xor(fl, o, 64);
        if (lane == 0) sh_f[wave] = fl;
        __syncthreads();
        fl = sh_f[0] | sh_f[1] | sh_f[2] | sh_f[3];
        if (tid == 0) lse[r] = (fl & 1) ? __int_as_float(0x7FC00000) : INFINITY;
    } else if (tid == 0) {
        lse[r] = Mref + logf(S);
    }
}

DD_DEV uint32_t verify_word(const VerifyArgs& a, int s, uint32_t stream, int idx, int explicit_off) {
    if (a.noise) return a.noise[(int64_t)s * a.nu + explicit_off + idx];
    return counter_word(a.seed, stream, a.step, a.row0 + (uint32_t)s, (uint32_t)idx);
}

DD_DEV float word_uniform_f(uint32_t w) { return ((float)w + 0.5f) * 0x1p-32f; }

template <typename T>
__global__ __launch_bounds__(VT) void verify_kernel(VerifyArgs a, const float* lse) {
    extern __shared__ float s_mass[];   // one mass per group
    __shared__ int sh_n;
    __shared__ float sh_tot[VT / 64];
    constexpr int E = Elem<T>::E;
    constexpr int LPG = DD_GUMBEL_GROUP / E;   // chunks (lanes) per group
    const int s = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
    const int B = a.B, V = a.V;
    const int ngroups = (V + DD_GUMBEL_GROUP - 1) / DD_GUMBEL_GROUP;
    const float* lse_p = lse + (size_t)s * B;
    const float* lse_q = lse + (size_t)a.S * B + (size_t)s * (B - 1);
    auto prow = [&](int i) { return (const char*)a.p + ((size_t)s * B + i) * a.ld * sizeof(T); };
    auto qrow = [&](int i) { return (const char*)a.q + ((size_t)s * (B - 1) + i) * a.ld * sizeof(T); };

    // ---- acceptance: the first rejected draft position (1-based), or B ----
    if (tid == 0) {
        int n = B;
        for (int i = 0; i < B - 1; ++i) {
            int x = a.draft[(int64_t)s * (B - 1) + i];
            if (x < 0 || x >= V) {
                if (a.err) atomicOr(a.err, DD_DEVERR_TOKEN);
                x = x < 0 ? 0 : V - 1;
            }
            const float lp = Elem<T>::load1(prow(i), x) - lse_p[i];
            const float lq = Elem<T>::load1(qrow(i), x) - lse_q[i];
            const float ratio = fminf(1.f, __builtin_amdgcn_exp2f((lp - lq) * LOG2E));
            const float u = word_uniform_f(verify_word(a, s, STREAM_VERIFY, i, 0));
            if (u > ratio) { n = i + 1; break; }
        }
        sh_n = n;
    }
    __syncthreads();
    const int n = sh_n;
    const bool resid = n < B;
    const char* pr = prow(n - 1);
    const char* qr = resid ? qrow(n - 1) : nullptr;
    const float lp0 = lse_p[n - 1], lq0 = resid ? lse_q[n - 1] : 0.f;

    // unnormalised class mass: [p - q]_+ for a rejection, p for the bonus (use_p: residual empty)
    auto cls_mass = [&](float lpv, float lqv, bool use_p) -> float {
        const float ep = __builtin_amdgcn_exp2f((lpv - lp0) * LOG2E);
        if (!resid || use_p) return ep;
        return fmaxf(ep - __builtin_amdgcn_exp2f((lqv - lq0) * LOG2E), 0.f);
    };

    // ---- group masses: lanes of a group hold consecutive chunks; reduce over LPG lanes ----
    const int nchunk = (V + E - 1) / E;
    auto masses = [&](bool use_p) -> float {
        float tot = 0.f;
        for (int c0 = 0; c0 < nchunk; c0 += VT) {
            const int c = c0 + tid;
            float sum = 0.f;
            if (c < nchunk) {
                const uint4 xp = *(const uint4*)(pr + (size_t)c * 16);
                uint4 xq = make_uint4(0u, 0u, 0u, 0u);
                if (resid && !use_p) xq = *(const uint4*)(qr + (size_t)c * 16);
#pragma unroll
                for (int e = 0; e < E; ++e)
                    if (c * E + e < V) sum += cls_mass(Elem<T>::get(xp, e), Elem<T>::get(xq, e), use_p);
            }
#pragma unroll
            for (int o = 1; o < LPG; o <<= 1) sum += __shfl_xor(sum, o, 64);
            if ((lane & (LPG - 1)) == 0 && c < nchunk) s_mass[c / LPG] = sum;
            tot += ((lane & (LPG - 1)) == 0 && c < nchunk) ? sum : 0.f;
        }
        tot = wave_sum(tot);
        if (lane == 0) sh_tot[tid >> 6] = tot;
        __syncthreads();
        float t = 0.f;
#pragma unroll
        for (int w = 0; w < VT / 64; ++w) t += sh_tot[w];
        __syncthreads();
        return t;
    };
    bool use_p = false;
    if (!(masses(false) > 0.f)) {   // empty residual: draw from p_n
        use_p = true;
        masses(true);
    }

    // ---- two-level draw (one wavefront) ----
    if ((tid >> 6) != 0) return;
    float best = -INFINITY;
    int bi = 0x7FFFFFFF;
    for (int g = lane; g < ngroups; g += 64) {
        const float sc = logf(s_mass[g]) + word_gumbel_f(verify_word(a, s, STREAM_TOP, g, B - 1));
        const bool take = sc > best || (sc == best && g < bi);
        best = take ? sc : best;
        bi = take ? g : bi;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float s2 = __shfl_xor(best, o, 64);
        const int i2 = __shfl_xor(bi, o, 64);
        const bool take = s2 > best || (s2 == best && i2 < bi);
        best = take ? s2 : best;
        bi = take ? i2 : bi;
    }
    const int gstar = bi;
    // no group with a valid score (NaN or +inf logits): report, emit token 0, index nothing
    const bool bad = gstar >= ngroups || !isfinite(lp0) || (resid && !use_p && !isfinite(lq0));
    best = -INFINITY;
    bi = 0x7FFFFFFF;
    const int ntop = ngroups;
    const int jend = bad ? 0 : min(V, (gstar + 1) * DD_GUMBEL_GROUP);
    for (int j = bad ? 0 : gstar * DD_GUMBEL_GROUP + lane; j < jend; j += 64) {
        const float lpv = Elem<T>::load1(pr, j);
        const float lqv = (resid && !use_p) ? Elem<T>::load1(qr, j) : 0.f;
        const float sc = logf(cls_mass(lpv, lqv, use_p)) +
                         word_gumbel_f(verify_word(a, s, STREAM_CLASS, j, B - 1 + ntop));
        const bool take = sc > best || (sc == best && j < bi);
        best = take ? sc : best;
        bi = take ? j : bi;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float s2 = __shfl_xor(best, o, 64);
        const int i2 = __shfl_xor(bi, o, 64);
        const bool take = s2 > best || (s2 == best && i2 < bi);
        best = take ? s2 : best;
        bi = take ? i2 : bi;
    }
    const bool bad_z = bad || bi >= V;
    if (lane == 0) {
        if (bad_z && a.err) atomicOr(a.err, DD_DEVERR_LOGITS);
        a.n_out[s] = n;
        a.z_out[s] = bad_z ? 0 : bi;
    }
}

}  // namespace

// Row log-sum-exps of dd_spec_verify_noalloc: a file-scope device array instead of a caller
// workspace, one copy per device, held until the process ends.  In host code `scratch` names a
// host-side stand-in, not device memory: the host takes each device's address from
// hipGetSymbolAddress (once per device, with that device current) and passes that address on.
static __device__ __align__(256) float scratch[DD_SPEC_VERIFY_NOALLOC_ROWS];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static float* g_scratch_dev[kMaxDevices] = {};

dd_status verify_noalloc_scratch(float** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        set_error("spec_verify_noalloc: hipGetDevice: %s", hipGetErrorString(e));
        return DD_E_HIP;
    }
    if (dev < 0 || dev >= kMaxDevices) {
        set_error("spec_verify_noalloc: device %d beyond the %d this library tracks", dev, kMaxDevices);
        return DD_E_UNSUPPORTED;
    }
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            set_error("spec_verify_noalloc: hipGetSymbolAddress: %s", hipGetErrorString(e));
            return DD_E_HIP;
        }
        g_scratch_dev[dev] = (float*)p;
    }
    *out = g_scratch_dev[dev];
    return DD_OK;
}

dd_status launch_verify(const VerifyArgs& a, int logits_dtype, float* lse, hipStream_t s) {
    if (a.S == 0) return DD_OK;
    const int rows = a.S * (2 * a.B - 1);
    const int ngroups = (a.V + DD_GUMBEL_GROUP - 1) / DD_GUMBEL_GROUP;
    const size_t shmem = (size_t)ngroups * sizeof(float);
    if (logits_dtype == DD_BF16) {
        launch_k(row_lse_kernel<bf16_t>, dim3(rows), dim3(VT), 0, s, a, lse);
        launch_k(verify_kernel<bf16_t>, dim3(a.S), dim3(VT), shmem, s, a, (const float*)lse);
    } else {
        launch_k(row_lse_kernel<float>, dim3(rows), dim3(VT), 0, s, a, lse);
        launch_k(verify_kernel<float>, dim3(a.S), dim3(VT), shmem, s, a, (const float*)lse);
    }
    return launch_status("spec_verify");
}

}  // namespace dd
