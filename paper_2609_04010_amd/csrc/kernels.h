// Argument blocks and launchers shared by the host code (dd_api.hip) and the kernel files.
#pragma once

#include "common.h"

namespace dd {

struct PostArgs {
    const void* logits;
    int64_t ld;
    int32_t rows, V, prior;
    const int32_t* z_t;
    int32_t* z_s;
    // masked prior, masked rows: p_v = w_x x_v, p_mask = w_m (stage 0 of the draw), log w_x
    double log_wx, wx, wm;
    // masked prior, unmasked rows under a Psi transition with kappa < 1: keep the token with
    // probability keep, remask with probability rmask (remask != 0 when rmask > 0)
    double keep, rmask;
    int32_t remask;
    // uniform prior: p_j = (c_x x_j + c_u + u1 D + [j == r](Ka_r x_r + c_z)) / D,
    // D = Ka_t x_r + one_m_at
    double c_x, c_u, u1, c_z, Ka_t, Ka_r, one_m_at;
    const uint32_t* noise;  // explicit words [rows][nu] or NULL (Philox)
    int32_t nu, ntop;
    uint64_t seed;
    uint32_t step, row0;
    float* probs;
    int32_t* err;
    // compacted mode (masked prior): logits row j belongs to token row rows_idx[j], j < *count
    const int32_t* rows_idx;
    const int32_t* count;
    // per-group log-sum-exps of the logits rows, [rows][glse_ld] (written by the vocabulary
    // projection's EPI_LSE epilogue), or NULL: then the posterior kernel computes them itself
    const float* glse;
    int64_t glse_ld;
    // with glse: each row's per-group level-2 candidates [rows][cand_ld] (EPI_LSE_CDF), or NULL: then
    // level 2 reads the chosen group's logits (masked prior only)
    const int32_t* cand;
    int64_t cand_ld;
    // per token row drawn: the log-sum-exp of its V logits as the draw computes it (or NULL)
    float* row_lse;
};

// EPI_GATE: C = bf16(acc * s_m), s_m = gate_scale if gate is NULL or gate[m % gate_period] != 0,
// else 0 (the adapter down-projection of a gated LoRA, written beside its input)
// EPI_LSE: plain bf16 store, and per row the log-sum-exp of each DD_GUMBEL_GROUP-column group of
// the stored (rounded) values into lse[m * lse_ld + n / DD_GUMBEL_GROUP] (vocabulary projection
// feeding the sampler; bf16, K % 128 == 0, 256-column tiles)
// EPI_LSE_CDF: EPI_LSE without storing the logits; instead, per row and group, the group's
// inverse-CDF candidate: the first class whose running sum of exp(l - ref) over the group exceeds
// u times the group's sum, u the Philox uniform of word (group, row0 + token row, step,
// STREAM_GROUP_U), into cand[m * cand_ld + n / DD_GUMBEL_GROUP] (the level 2 of the store-free
// two-level draw)
enum Epi { EPI_BIAS = 0, EPI_BIAS_GELU = 1, EPI_BIAS_RESID = 2, EPI_PLAIN = 3, EPI_GATE = 4, EPI_LSE = 5,
           EPI_LSE_CDF = 6 };

struct GemmArgs {
    const void* A;   // [M][K], row stride lda
    int64_t lda;
    const void* W;   // [N][K], row stride ldw
    int64_t ldw;
    const void* bias;
    void* C;         // [M][N], row stride ldc
    int64_t ldc;
    int M, N, K;
    // optional row gather (bf16 path, K % 64 == 0): output row m < *m_count takes A row a_rows[m]
    const int32_t* a_rows;
    const int32_t* m_count;
    // EPI_GATE only: per-row gate, read at m % gate_period, and the scale of open rows
    const int32_t* gate;
    int gate_period;
    float gate_scale;
    // EPI_LSE / EPI_LSE_CDF: group log-sum-exps [M][lse_ld]
    float* lse;
    int64_t lse_ld;
    // EPI_LSE_CDF only: group candidates [M][cand_ld]; the noise key and counters (the token row of
    // output row m is a_rows[m] when gathered, else m)
    int32_t* cand;
    int64_t cand_ld;
    uint64_t seed;
    uint32_t step, row0;
    // EPI_BIAS_RESID, bf16 path: the residual input when it is not C itself.  Output row m of C
    // then adds row c_rows[m] of c_in (row m when c_rows is NULL); both have row stride ldc.
    const float* c_in;
    const int32_t* c_rows;
    // EPI_LSE_CDF: token row of output row m when A is already compacted (takes precedence over
    // a_rows for the noise counters)
    const int32_t* row_ids;
    // tile_hint k > 0: use tile shape k - 1 of the launcher's table (0: chosen from the shape)
    int tile_hint;
    // m_gate > 0 (with m_count): the launch does its work only if *m_count > m_gate (m_side 0)
    // or *m_count <= m_gate (m_side 1); two launches with the two sides pick a tile shape by the
    // device-side row count
    int m_gate, m_side;
};

struct AttnArgs {
    const void* qkv;  // [B*L][3d]: q | k | v, head h at columns h*dh
    int64_t ld;
    void* out;        // [B*L][d]
    int64_t ldo;
    int B, L, H, d;
    float scale_log2;  // log2(e) / sqrt(dh)
    // visibility (NULL: every key): key j is visible to query i iff j < pre[i] or lo[i] <= j < hi[i],
    // with pre = mask[0..L), lo = mask[L..2L), hi = mask[2L..3L); an entry outside 0 <= pre <= L,
    // 0 <= lo <= hi <= L, or with no visible key, sets DD_DEVERR_MASK in *err and sees every key
    const int32_t* mask;
    int32_t* err;
    int hgroup;   // set by launch_attn: (batch, head) pairs per dispatch group of the pattern kernel
    // listed queries only (bf16, no pattern; nullable): qrows is a row list sorted by row, qseq[b]
    // the index in it of sequence b's first row (qseq[B] = its length).  Output row j is the query
    // at token row qrows[j]; every key of its sequence is still visible.
    const int32_t* qrows;
    const int32_t* qseq;
};

dd_status launch_posterior(const PostArgs& a, int logits_dtype, hipStream_t s);
// keep-or-remask draw of every unmasked row (masked prior, kappa < 1), one thread per row
dd_status launch_remask(const PostArgs& a, hipStream_t s);

// Speculative verification: target rows p [S*B][ld], draft rows q [S*(B-1)][ld], drafted tokens
// [S][B-1]; outputs n (first rejected position, 1-based, or B) and the replacement / bonus token.
struct VerifyArgs {
    const void* p;
    const void* q;
    int64_t ld;
    int32_t S, B, V;
    const int32_t* draft;
    const uint32_t* noise;  // explicit words [S][nu] or NULL (Philox)
    int32_t nu;
    uint64_t seed;
    uint32_t step, row0;
    int32_t* n_out;
    int32_t* z_out;
    int32_t* err;
};
dd_status launch_verify(const VerifyArgs& a, int logits_dtype, float* lse, hipStream_t s);
// Device address of the current device's DD_SPEC_VERIFY_NOALLOC_ROWS-float array of
// dd_spec_verify_noalloc (looked up on the first call on each device).
dd_status verify_noalloc_scratch(float** out);
dd_status launch_latent(const int32_t* x, int32_t rows, int32_t V, double at, double sigma,
                        uint64_t seed, uint32_t step, uint32_t row0, int32_t* z, int32_t* err,
                        hipStream_t s);
dd_status launch_init(void* dst, int64_t count, uint32_t id, double shift, int is_bf16,
                      uint64_t seed, hipStream_t s);
dd_status launch_temb(float* temb, int d, double tau, hipStream_t s);
// norm: dd_norm (LayerNorm or RMSNorm; b is not read under RMSNorm)
dd_status launch_embed_ln(int dtype, int norm, const int32_t* z, int64_t rows, int L, int n_tok, int d,
                          const void* tok, const void* pos, const float* temb, const void* g,
                          const void* b, float eps, float* h, void* xln, int64_t ldo, int32_t* err,
                          hipStream_t s);
// out rows have stride ldo (elements) >= d
// m_count (device, nullable): only rows < *m_count are normalised (rows bounds the grid)
dd_status launch_ln(int dtype, int norm, const float* h, int64_t rows, int d, const void* g, const void* b,
                    float eps, void* out, int64_t ldo, hipStream_t s, const int32_t* m_count = nullptr);
bool ln_supported(int d);
dd_status launch_gemm(int dtype, int epi, int cls, const GemmArgs& g, hipStream_t s);
dd_status launch_attn(int dtype, const AttnArgs& a, hipStream_t s);
bool attn_supported(int dtype, int dh);
// seq (device, nullable): seq[b] = listed rows before row b L for b = 0..M/L (rows of L tokens).
// pre (host, nullable; masked prior): list only the masked rows that stage 0 of the draw described
// by *pre unmasks (the others stay masked and need no logits)
dd_status launch_compact(const int32_t* z, int64_t M, int32_t mask_id, int32_t* idx, int32_t* count,
                         hipStream_t s, int L = 0, int32_t* seq = nullptr, const PostArgs* pre = nullptr);
bool gemm_gather_supported(int dtype, int K);
// the EPI_LSE epilogue (group log-sum-exps beside the logits) runs for this dtype and K
bool gemm_lse_supported(int dtype, int K);

}  // namespace dd
