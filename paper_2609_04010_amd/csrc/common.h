// Shared device/host helpers of the gfx950 reverse-step library.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <tuple>

#include "dd.h"

#define DD_DEV __device__ __forceinline__

typedef uint16_t bf16_t;  // raw bfloat16 bits

// ---------------------------------------------------------------- bf16 <-> fp32
DD_DEV float bf16_lo(uint32_t pair) { return __uint_as_float(pair << 16); }
DD_DEV float bf16_hi(uint32_t pair) { return __uint_as_float(pair & 0xFFFF0000u); }
DD_DEV float bf16_to_f32(bf16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// Round-to-nearest-even fp32 -> bf16 with the hardware conversion (v_cvt_pk_bf16_f32, which rounds
// in the default round-to-nearest-even mode).
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_hw;
DD_DEV uint32_t pack_bf16x2(float lo, float hi) {
    const bf16x2_hw v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
}
DD_DEV bf16_t f32_to_bf16(float f) { return (bf16_t)(pack_bf16x2(f, 0.f) & 0xFFFFu); }

// Round-to-nearest-even float64 -> bf16 directly (no intermediate fp32 rounding).
DD_DEV bf16_t f64_to_bf16(double v) {
    uint64_t b = (uint64_t)__double_as_longlong(v);
    uint32_t sign = (uint32_t)(b >> 63);
    uint64_t mag = b & 0x7FFFFFFFFFFFFFFFull;
    if (mag == 0) return (bf16_t)(sign << 15);
    // keep 7 mantissa bits of 52: round at bit 45, ties to even
    uint64_t lsb = (mag >> 45) & 1ull;
    mag += (1ull << 44) - 1ull + lsb;
    int32_t e11 = (int32_t)(mag >> 52);
    uint32_t m7 = (uint32_t)((mag >> 45) & 0x7Full);
    int32_t e8 = e11 - 1023 + 127;
    if (e8 <= 0) return (bf16_t)(sign << 15);           // below bf16 normals: flush
    if (e8 >= 255) return (bf16_t)((sign << 15) | 0x7F80u);
    return (bf16_t)((sign << 15) | ((uint32_t)e8 << 7) | m7);
}

// ---------------------------------------------------------------- wave helpers
DD_DEV float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}
// Wavefront sum with DPP lane moves (VALU latency, no LDS round trips): two quad permutations and
// the half-row and row mirrors leave every lane of a 16-lane row with that row's sum; the row
// broadcasts of lanes 15 and 31 then add rows 0 and 2 into rows 1 and 3 and rows 0-1 into rows 2-3
// (lanes outside a move's row mask add 0), so lane 63 ends with the total, which every lane gets.
template <int CTRL, int ROW_MASK>
DD_DEV float dpp_add(float v) {
    const int m = __builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROW_MASK, 0xF, false);
    return v + __int_as_float(m);
}
DD_DEV float wave_sum_dpp(float v) {
    v = dpp_add<0xB1, 0xF>(v);    // quad_perm [1, 0, 3, 2]
    v = dpp_add<0x4E, 0xF>(v);    // quad_perm [2, 3, 0, 1]
    v = dpp_add<0x141, 0xF>(v);   // row_half_mirror
    v = dpp_add<0x140, 0xF>(v);   // row_mirror
    v = dpp_add<0x142, 0xA>(v);   // row_bcast15 into rows 1 and 3
    v = dpp_add<0x143, 0xC>(v);   // row_bcast31 into rows 2 and 3
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}
DD_DEV float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}

// Workgroup id -> work index such that each of the 8 XCDs (which receive workgroups round-robin by
// id) walks one contiguous eighth of the work indices; work that shares operands and sits close in
// index order then shares that XCD's L2.  Ids past the largest multiple of 8 map to themselves.
DD_DEV int xcd_linear(int bid, int nblocks) {
    const int per = nblocks / 8;
    return bid < per * 8 ? (bid & 7) * per + (bid >> 3) : bid;
}

// ---------------------------------------------------------------- host helpers
namespace dd {

void set_error(const char* fmt, ...);
dd_status launch_status(const char* what);

// Profiling hooks around each launch (no-ops unless dd_profile_begin was called).
enum KernelClass {
    KC_TEMB = 0, KC_EMBED_LN, KC_LN, KC_GEMM_QKV, KC_ATTN, KC_GEMM_O, KC_GEMM_MLP1,
    KC_GEMM_MLP2, KC_GEMM_VOCAB, KC_POSTERIOR, KC_LATENT, KC_INIT, KC_COPY, KC_COMPACT, KC_GEMM_LORA,
    KC_COUNT
};
// A scope around one kernel launch (kernel = true) hands its event pair to that launch (launch_k),
// which records them as part of the dispatch (hipExtLaunchKernel): no marker packets of their own
// between the kernels.  Other scopes (a copy) record the events around their work.
void prof_start(int cls, hipStream_t s, bool kernel);
void prof_stop(int cls, hipStream_t s);
// the event pair a kernel-launch scope opened on this host thread (once; false if none)
bool prof_take(hipEvent_t* start, hipEvent_t* stop);

struct ProfScope {
    int cls;
    hipStream_t s;
    ProfScope(int c, hipStream_t st, bool kernel = true) : cls(c), s(st) { prof_start(cls, s, kernel); }
    ~ProfScope() { prof_stop(cls, s); }
};

// Launch of kernel k with its arguments converted to the kernel's parameter types; with the event
// pair of an enclosing profiling scope, through hipExtLaunchKernel.
template <typename... KP, typename... A>
inline void launch_k(void (*k)(KP...), dim3 grid, dim3 block, uint32_t shmem, hipStream_t s, A... a) {
    static_assert(sizeof...(KP) == sizeof...(A), "argument count");
    std::tuple<KP...> args(static_cast<KP>(a)...);
    std::apply(
        [&](auto&... x) {
            void* argv[] = {(void*)&x..., nullptr};
            hipEvent_t e0, e1;
            if (prof_take(&e0, &e1))
                (void)hipExtLaunchKernel((const void*)k, grid, block, argv, shmem, s, e0, e1, 0);
            else
                (void)hipLaunchKernel((const void*)k, grid, block, argv, shmem, s);
        },
        args);
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace dd
