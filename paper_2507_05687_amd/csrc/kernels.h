// Internal kernel launch interface of libgrpo (not part of the ABI).
#pragma once

#include "common.h"

namespace grpo {

// ---------------------------------------------------------------- GEMM
// C[m, n] = sum_k A[m, k] * B[n, k]; A and B bf16 in the tiled layout.
struct GemmArgs {
  const uint16_t* A;
  int M;                  // rows of A (static bound)
  const uint16_t* B;
  int N;                  // rows of B (static bound)
  const int32_t* m_dev;   // optional device bound on M (e.g. the valid-token count)
  const int32_t* n_dev;   // optional device bound on N
  // Operand storage (tiled layout, 256 x 32 blocks). A natural operand is
  // stored [rows = its M (or N)][columns = K]: x_kt blocks per block-row, K
  // starting at block x_kb0. A transposed operand is stored [rows = K]
  // [columns = its M (or N)]: x_kt blocks per block-row, K starting at row
  // 32 * x_kb0, its columns starting at block x_cb0.
  int64_t a_kt, a_kb0, a_cb0;
  int64_t b_kt, b_kb0, b_cb0;
  int K;                  // contraction length, a multiple of 32 (when k_dev is NULL)
  const int32_t* k_dev;   // optional device K, rounded up to 32 (operands zero-padded)
  int tiles_m, tiles_n;   // 256x256 tiles covering the static M x N
  int splits;             // K split over this many workgroups per tile (grid y), 1 = none
};

struct StoreArgs {
  float* acc_buf;
  int64_t ld_acc;
  int read_acc;
  void* out;
  int64_t ld_out;
  int out_bf16;
  int add_out;
  const int32_t* out_rows;
  int64_t m_limit;
  int64_t n_limit;
  int64_t split_stride;  // with a split K: elements between the splits' acc_buf partials
  // optional term added to every stored row m: oh_g[m] * row oh_y[m] of the bf16
  // matrix oh_w (row stride oh_ld); used only on the product that writes `out`
  const float* oh_g;
  const int32_t* oh_y;
  const uint16_t* oh_w;
  int64_t oh_ld;
};

int gemm_grid(int tiles_m, int tiles_n);
// scoring of the vocabulary rows [v0, v0 + g.M) (A = those rows of W); the
// partials of vocabulary tile i go to row i of ms
void launch_gemm_lse(const GemmArgs& g, const int32_t* y_p, float* zy, float2* ms, int64_t ldms,
                     int64_t V, int64_t v0, hipStream_t s);
// dz = -g * exp(z - lse) for a vocabulary chunk starting at row v0 (the
// sampled id's +g is left to the gradient products' callers)
void launch_gemm_dz(const GemmArgs& g, const float* lse_p, const float* g_p, uint16_t* dz,
                    int64_t dz_kt, int64_t V, int64_t v0, hipStream_t s);
void launch_gemm_store(const GemmArgs& g, const StoreArgs& a, bool grad_weight, hipStream_t s);

// ------------------------------------------------------------- packing
struct PackArgs {
  const uint8_t* mask;
  const int64_t* tokens;  // optional: ids are range-checked against V
  int64_t V;
  const int64_t* cu;
  int64_t seg;       // cu == NULL: rows are packed in segments of seg rows, B = their count
  int64_t B, N;
  int32_t* counts;   // [B]
  int32_t* base;     // [B+1]
  int32_t* rows_p;   // [N] packed -> row
  int32_t* seq_p;    // [N] packed -> rollout (optional)
  int32_t* y_p;      // [N] packed -> token id (optional)
  int32_t* pidx;     // [N] row -> packed or -1 (optional)
  int32_t* num_valid_out;  // optional extra copy of the count
  int64_t cap;             // more valid rows than this: err_capacity, and no row is valid
  WsHeader* hdr;
};
void launch_pack(const PackArgs& a, hipStream_t s);
// *out = the status code the header's error words stand for (0 if none)
void launch_copy_status(const WsHeader* hdr, int32_t* out, hipStream_t s);

// ------------------------------------------------ token objective (Eq. 1)
// objective 0: the GRPO surrogate of Eq. 1; objective 1: the supervised
// cross-entropy of the SFT stage (mean over valid tokens of -logp).
struct TokenArgs {
  int objective;
  int64_t N, B;
  const int32_t* pidx;
  const int32_t* seq_p;
  const int32_t* counts;
  const WsHeader* hdr;
  const float* adv;
  const float* logp_p;
  const float* lse_p;
  const float* old_logp;
  const float* ref_logp;
  float eps, beta;
  int agg;
  float* g_p;
  float* logp_out;
  float* lse_out;
  float* token_loss;
  float* dlogp;
  uint8_t* clip_flag;
  float* loss_part;
  float* loss;
};
int64_t token_objective_blocks(int64_t N);
void launch_token_objective(const TokenArgs& a, hipStream_t s);

// ------------------------------------------------ sampled-id term of dL/dW
// dW[y_t] += g_t h_t for every valid packed token t, summed per id in packed
// order (ids grouped by a stable radix sort). keys/vals: two int32 buffers of
// n each; counts: onehot_count_entries(n) int32.
struct OnehotArgs {
  const int32_t* y_p;     // packed token -> id
  const int32_t* rows_p;  // packed token -> row of hidden
  const float* g_p;       // packed token -> dL/dlogp
  const WsHeader* hdr;    // num_valid
  const uint16_t* hidden; // bf16 [rows][H], H % 8 == 0, 16-byte aligned
  int64_t H, V;
  int64_t n;              // packed rows covered (>= num_valid)
  int32_t* keys[2];
  int32_t* vals[2];
  int32_t* counts;
  float* dW;              // [V][H]
};
int64_t onehot_count_entries(int64_t n);
void launch_onehot_dw(const OnehotArgs& a, hipStream_t s);

// ------------------------------------------------------------ AdamW
struct AdamArgs {
  float* w;
  float* m;
  float* v;
  const float* g;
  uint16_t* w_bf16;  // optional
  int64_t n;
  float beta1, beta2, eps;
  float decay;         // 1 - lr * weight_decay
  float step_size;     // lr / (1 - beta1^t)
  float inv_sqrt_bc2;  // 1 / sqrt(1 - beta2^t)
};
void launch_adamw(const AdamArgs& a, hipStream_t s);
// dL/dh of packed row t < num_valid (rows of the grid: `rows`) into output row
// rows_p[t]: the split partials part[s * stride + t * ld + c] summed in split
// order, plus g_t W[y_t, c], rounded once (bf16 or fp32 output)
void launch_dh_finish(const float* part, int splits, int64_t stride, int64_t ld,
                      const WsHeader* hdr, int64_t rows, int64_t H, const float* g_p,
                      const int32_t* y_p, const uint16_t* W, const int32_t* rows_p, void* out,
                      int out_bf16, hipStream_t s);
// out[r, c] (+)= the sum over s < splits of part[s * stride + r * ld_part + c], summed in
// split order before it is added
void launch_sum_splits(const float* part, int splits, int64_t stride, int64_t ld_part, float* out,
                       int64_t ld_out, int64_t rows, int64_t cols, int accumulate, hipStream_t s);

// ------------------------------------------------------------ rule reward
struct RewardArgs {
  const uint8_t* text;         // completions, concatenated
  int64_t text_bytes;          // readable bytes at text
  const int64_t* offsets;      // [count + 1]; pairs outside [0, text_bytes] are empty
  const uint8_t* test_passed;  // [count]
  int require_launch;          // is_Triton also needs a launch of the kernel
  int weighted;                // reward = w_rule*is_Triton + w_exec*passed (else the product)
  float w_rule, w_exec;
  uint8_t* is_triton;  // [count]
  float* reward;       // [count]
};
void launch_rule_reward(const RewardArgs& a, int64_t count, hipStream_t s);

// ------------------------------------------------------------ others
void launch_group_advantages(const float* rewards, int64_t num_prompts, int group, float eps,
                             int unbiased, float* adv, hipStream_t s);
void launch_lse_finalize(const float2* ms, int64_t ldms, int tiles, const float* zy,
                         const WsHeader* hdr, float* lse_p, float* logp_p, int64_t Nmax,
                         hipStream_t s);
void launch_logp_from_lse(const float* zy, const float* lse_in, const int32_t* rows_p,
                          const WsHeader* hdr, float* lse_p, float* logp_p, int64_t Nmax,
                          hipStream_t s);
void launch_rows_out(const int32_t* pidx, int64_t N, const float* logp_p, const float* lse_p,
                     float* logp, float* lse, hipStream_t s);
void launch_gather_dot_bf16(const uint16_t* hidden, const uint16_t* W, int64_t H,
                            const int32_t* rows_p, const int32_t* y_p, const WsHeader* hdr,
                            float* zy, int64_t Nmax, hipStream_t s);
// Tiled layout of rows of `in` (row i = in[rows ? rows[i] : i], K columns):
// r_pad x round_up(K, 32), rows >= the valid count (hdr->num_valid, else
// n_static) and columns >= K zero; tile-rows `stride` blocks apart.
void launch_tile_rows(const uint16_t* in, int64_t ld_in, const int32_t* rows, int64_t n_static,
                      const WsHeader* hdr, int64_t r_pad, int64_t K, int64_t stride,
                      uint16_t* out, hipStream_t s);
void launch_zero_masked_rows(const int32_t* pidx, int64_t N, int64_t H, void* out, int out_bf16,
                             hipStream_t s);
void launch_f32_score(const float* hidden, const float* W, int64_t H, int64_t V,
                      const int32_t* rows_p, const int32_t* y_p, const WsHeader* hdr,
                      float* lse_p, float* logp_p, float* zy_p, int64_t Nmax, hipStream_t s);
void launch_f32_grad_hidden(const float* hidden, const float* W, int64_t H, int64_t V,
                            const int32_t* rows_p, const int32_t* y_p, const float* lse_p,
                            const float* g_p, const WsHeader* hdr, float* grad_hidden,
                            int64_t Nmax, hipStream_t s);
void launch_f32_grad_weight(const float* hidden, const float* W, int64_t H, int64_t V,
                            const int32_t* rows_p, const int32_t* y_p, const float* lse_p,
                            const float* g_p, const WsHeader* hdr, float* grad_weight,
                            int accumulate, hipStream_t s);

}  // namespace grpo
