// Streaming and bookkeeping kernels of libgrpo: group advantages (Eq. 2),
// valid-row packing (the |o_i| counts of Eq. 1), the per-token GRPO term
// (Eq. 1), the log-sum-exp combine, operand tiling, and the plain fp32 path.
//
// All reductions run in a fixed order, so every result is bitwise
// reproducible run to run. No kernel uses atomics.
#include "kernels.h"

#include <math.h>

namespace grpo {

// ------------------------------------------------------------- helpers
__device__ inline float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}
__device__ inline float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ inline float wave_min(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fminf(x, __shfl_xor(x, o, 64));
  return x;
}

// Sum over a 256-thread block, same association for every call.
__device__ inline float block_sum_256(float x, float* red /*[4]*/) {
  x = wave_sum(x);
  int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = x;
  __syncthreads();
  float t = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return t;
}

// Online (max, sum-exp) merge; an empty partial is (-inf, 0).
__device__ inline void lse_merge(float& m, float& s, float m2, float s2) {
  if (s2 == 0.f) return;
  if (s == 0.f) { m = m2; s = s2; return; }
  if (m2 > m) { s = s * __expf(m - m2) + s2; m = m2; }
  else { s += s2 * __expf(m2 - m); }
}

// ---------------------------------------------------- Eq. 2 advantages
// One wave per prompt group. Two passes over the group's rewards: range and
// mean, then the squared deviations.
__global__ void __launch_bounds__(256) k_group_advantages(const float* __restrict__ rewards,
                                                           int64_t num_prompts, int group,
                                                           float eps, int unbiased,
                                                           float* __restrict__ adv) {
  int64_t p = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  int lane = threadIdx.x & 63;
  if (p >= num_prompts) return;
  const float* r = rewards + p * group;
  float* a = adv + p * group;
  float lo = INFINITY, hi = -INFINITY, sum = 0.f;
  for (int i = lane; i < group; i += 64) {
    float v = r[i];
    lo = fminf(lo, v);
    hi = fmaxf(hi, v);
    sum += v;
  }
  lo = wave_min(lo);
  hi = wave_max(hi);
  if (lo == hi) {  // all-equal group: exactly zero
    for (int i = lane; i < group; i += 64) a[i] = 0.f;
    return;
  }
  float mean = wave_sum(sum) / (float)group;
  float ss = 0.f;
  for (int i = lane; i < group; i += 64) {
    float d = r[i] - mean;
    ss += d * d;
  }
  ss = wave_sum(ss);
  float sd = sqrtf(ss / (float)(unbiased ? group - 1 : group));
  float inv = 1.f / (sd + eps);
  for (int i = lane; i < group; i += 64) a[i] = (r[i] - mean) * inv;
}

void launch_group_advantages(const float* rewards, int64_t num_prompts, int group, float eps,
                             int unbiased, float* adv, hipStream_t s) {
  int blocks = (int)ceil_div(num_prompts, 4);
  hipLaunchKernelGGL(k_group_advantages, dim3(blocks), dim3(256), 0, s, rewards, num_prompts,
                     group, eps, unbiased, adv);
}

// ------------------------------------------------------- row packing
__device__ inline bool row_valid(const uint8_t* mask, const int64_t* tokens, int64_t V, int64_t r,
                                 WsHeader* hdr) {
  if (mask && !mask[r]) return false;
  if (tokens) {
    int64_t y = tokens[r];
    if (y < 0 || y >= V) {
      hdr->err_token = 1;
      return false;
    }
  }
  return true;
}

// Row range of rollout b, checked against 0 = cu[0] <= ... <= cu[B] = N.
// cu == NULL stands for a single rollout covering every row, cut into
// segments of `seg` rows (one workgroup each); b is then a segment.
__device__ inline bool seq_range(const int64_t* cu, int64_t seg, int64_t b, int64_t B, int64_t N,
                                 int64_t& lo, int64_t& hi, WsHeader* hdr) {
  if (cu == nullptr) {
    lo = b * seg;
    hi = lo + seg < N ? lo + seg : N;
    return true;
  }
  lo = cu[b];
  hi = cu[b + 1];
  bool ok = lo >= 0 && hi >= lo && hi <= N && (b != 0 || lo == 0) && (b != B - 1 || hi == N);
  if (!ok) {
    hdr->err_seqlens = 1;
    lo = hi = 0;
  }
  return ok;
}

__global__ void k_fill_i32(int32_t* p, int64_t n, int32_t v) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// counts[b] = number of valid rows of rollout b.
__global__ void __launch_bounds__(256) k_pack_count(const uint8_t* __restrict__ mask,
                                                    const int64_t* __restrict__ tokens, int64_t V,
                                                    const int64_t* __restrict__ cu, int64_t seg,
                                                    int64_t B, int64_t N,
                                                    int32_t* __restrict__ counts, WsHeader* hdr) {
  int64_t b = blockIdx.x;
  int64_t lo, hi;
  seq_range(cu, seg, b, B, N, lo, hi, hdr);
  int c = 0;
  for (int64_t r = lo + threadIdx.x; r < hi; r += 256) c += row_valid(mask, tokens, V, r, hdr);
  __shared__ int redi[256];
  redi[threadIdx.x] = c;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) redi[threadIdx.x] += redi[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) counts[b] = redi[0];
}

// Exclusive scan of counts -> base[b]; base[B] and hdr->num_valid = total.
__global__ void __launch_bounds__(256) k_pack_scan(const int32_t* __restrict__ counts, int64_t B,
                                                   int32_t* __restrict__ base, WsHeader* hdr,
                                                   int32_t* num_valid_out, int64_t cap) {
  __shared__ int32_t part[256];
  // each thread scans a contiguous slice
  int64_t per = ceil_div(B, 256);
  int64_t lo = threadIdx.x * per, hi = lo + per < B ? lo + per : B;
  int32_t s = 0;
  for (int64_t i = lo; i < hi; ++i) s += counts[i];
  part[threadIdx.x] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t run = 0;
    for (int i = 0; i < 256; ++i) {
      int32_t t = part[i];
      part[i] = run;
      run += t;
    }
    if (run > cap) {  // the workspace holds fewer rows: the call counts none as valid
      hdr->err_capacity = 1;
      run = 0;
    }
    hdr->num_valid = run;
    base[B] = run;
    if (num_valid_out) *num_valid_out = run;
  }
  __syncthreads();
  int32_t run = part[threadIdx.x];
  for (int64_t i = lo; i < hi; ++i) {
    base[i] = run;
    run += counts[i];
  }
}

// Writes, for rollout b, the packed position of each of its valid rows:
// rows_p[j] = row, seq_p[j] = b, y_p[j] = token id, pidx[row] = j (or -1).
__global__ void __launch_bounds__(256) k_pack_scatter(
    const uint8_t* __restrict__ mask, const int64_t* __restrict__ tokens, int64_t V,
    const int64_t* __restrict__ cu, int64_t seg, int64_t B, int64_t N,
    const int32_t* __restrict__ base,
    int32_t* __restrict__ rows_p, int32_t* __restrict__ seq_p, int32_t* __restrict__ y_p,
    int32_t* __restrict__ pidx, WsHeader* hdr) {
  __shared__ int32_t wcount[4];
  int64_t b = blockIdx.x;
  int64_t lo, hi;
  seq_range(cu, seg, b, B, N, lo, hi, hdr);
  int32_t next = base[b];
  int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (hdr->err_capacity) return;  // no row is valid (pidx stays -1)
  for (int64_t r0 = lo; r0 < hi; r0 += 256) {
    int64_t r = r0 + threadIdx.x;
    bool v = r < hi && row_valid(mask, tokens, V, r, hdr);
    uint64_t bal = __ballot(v);
    int below = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) wcount[w] = __popcll(bal);
    __syncthreads();
    int off = 0;
    for (int i = 0; i < w; ++i) off += wcount[i];
    int tot = wcount[0] + wcount[1] + wcount[2] + wcount[3];
    if (r < hi) {
      if (v) {
        int32_t j = next + off + below;
        if (rows_p) rows_p[j] = (int32_t)r;
        if (seq_p) seq_p[j] = (int32_t)b;
        if (y_p) y_p[j] = (int32_t)tokens[r];
        if (pidx) pidx[r] = j;
      } else if (pidx) {
        pidx[r] = -1;
      }
    }
    next += tot;
    __syncthreads();
  }
}

// Every entry point starts by clearing the workspace's error words, so that
// grpo_check_error() reports the most recent call on that workspace.
__global__ void k_reset_flags(WsHeader* hdr) {
  hdr->err_token = 0;
  hdr->err_seqlens = 0;
  hdr->err_capacity = 0;
}

// status of the most recent call on the workspace header: GRPO_ERR_SEQLENS
// (10), GRPO_ERR_TOKEN_RANGE (9) or 0
__global__ void k_copy_status(const WsHeader* hdr, int32_t* out) {
  *out = hdr->err_seqlens ? 10 : hdr->err_token ? 9 : hdr->err_capacity ? 11 : 0;
}

void launch_copy_status(const WsHeader* hdr, int32_t* out, hipStream_t s) {
  hipLaunchKernelGGL(k_copy_status, dim3(1), dim3(1), 0, s, hdr, out);
}

void launch_pack(const PackArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_reset_flags, dim3(1), dim3(1), 0, s, a.hdr);
  if (a.pidx) {
    hipLaunchKernelGGL(k_fill_i32, dim3((unsigned)ceil_div(a.N, 256)), dim3(256), 0, s, a.pidx,
                       a.N, -1);
  }
  hipLaunchKernelGGL(k_pack_count, dim3((unsigned)a.B), dim3(256), 0, s, a.mask, a.tokens, a.V,
                     a.cu, a.seg, a.B, a.N, a.counts, a.hdr);
  hipLaunchKernelGGL(k_pack_scan, dim3(1), dim3(256), 0, s, a.counts, a.B, a.base, a.hdr,
                     a.num_valid_out, a.cap);
  hipLaunchKernelGGL(k_pack_scatter, dim3((unsigned)a.B), dim3(256), 0, s, a.mask, a.tokens,
                     a.V, a.cu, a.seg, a.B, a.N, a.base, a.rows_p, a.seq_p, a.y_p, a.pidx, a.hdr);
}

// ------------------------------------------------------ lse combine
// lse of packed token j from the per-vocabulary-tile partials, then
// logp = z_y - lse. One token per lane (the partials of consecutive tokens are
// contiguous); the partials are merged in kChains interleaved chains, partial
// t going to chain t % kChains, so that that many loads are in flight, and the
// chains are then merged pairwise in a fixed order.
constexpr int kChains = 8;
__global__ void __launch_bounds__(64) k_lse_finalize(const float2* __restrict__ ms, int64_t ldms,
                                                     int tiles, const float* __restrict__ zy,
                                                     const WsHeader* __restrict__ hdr,
                                                     float* __restrict__ lse_p,
                                                     float* __restrict__ logp_p) {
  int64_t j = (int64_t)blockIdx.x * 64 + threadIdx.x;
  if (j >= hdr->num_valid) return;
  float m[kChains], s[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) {
    m[c] = -INFINITY;
    s[c] = 0.f;
  }
  int t = 0;
  for (; t + kChains <= tiles; t += kChains) {
    float2 p[kChains];
#pragma unroll
    for (int c = 0; c < kChains; ++c) p[c] = ms[(int64_t)(t + c) * ldms + j];
#pragma unroll
    for (int c = 0; c < kChains; ++c) lse_merge(m[c], s[c], p[c].x, p[c].y);
  }
#pragma unroll
  for (int c = 0; c < kChains - 1; ++c) {
    if (t + c < tiles) {
      const float2 p = ms[(int64_t)(t + c) * ldms + j];
      lse_merge(m[c], s[c], p.x, p.y);
    }
  }
#pragma unroll
  for (int w = 1; w < kChains; w *= 2)
#pragma unroll
    for (int c = 0; c + w < kChains; c += 2 * w) lse_merge(m[c], s[c], m[c + w], s[c + w]);
  float l = m[0] + __logf(s[0]);
  lse_p[j] = l;
  logp_p[j] = zy[j] - l;
}

void launch_lse_finalize(const float2* ms, int64_t ldms, int tiles, const float* zy,
                         const WsHeader* hdr, float* lse_p, float* logp_p, int64_t Nmax,
                         hipStream_t s) {
  hipLaunchKernelGGL(k_lse_finalize, dim3((unsigned)ceil_div(Nmax, 64)), dim3(64), 0, s, ms,
                     ldms, tiles, zy, hdr, lse_p, logp_p);
}

// With a caller-supplied lse: logp = z_y - lse_in[row].
__global__ void __launch_bounds__(256) k_logp_from_lse(const float* __restrict__ zy,
                                                       const float* __restrict__ lse_in,
                                                       const int32_t* __restrict__ rows_p,
                                                       const WsHeader* __restrict__ hdr,
                                                       float* __restrict__ lse_p,
                                                       float* __restrict__ logp_p) {
  int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j >= hdr->num_valid) return;
  float l = lse_in[rows_p[j]];
  lse_p[j] = l;
  logp_p[j] = zy[j] - l;
}

void launch_logp_from_lse(const float* zy, const float* lse_in, const int32_t* rows_p,
                          const WsHeader* hdr, float* lse_p, float* logp_p, int64_t Nmax,
                          hipStream_t s) {
  hipLaunchKernelGGL(k_logp_from_lse, dim3((unsigned)ceil_div(Nmax, 256)), dim3(256), 0, s, zy,
                     lse_in, rows_p, hdr, lse_p, logp_p);
}

// Scatter packed logp/lse to per-row outputs (0 on masked rows).
__global__ void __launch_bounds__(256) k_rows_out(const int32_t* __restrict__ pidx, int64_t N,
                                                  const float* __restrict__ logp_p,
                                                  const float* __restrict__ lse_p,
                                                  float* __restrict__ logp,
                                                  float* __restrict__ lse) {
  int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (r >= N) return;
  int32_t j = pidx[r];
  if (logp) logp[r] = j >= 0 ? logp_p[j] : 0.f;
  if (lse) lse[r] = j >= 0 ? lse_p[j] : 0.f;
}

void launch_rows_out(const int32_t* pidx, int64_t N, const float* logp_p, const float* lse_p,
                     float* logp, float* lse, hipStream_t s) {
  hipLaunchKernelGGL(k_rows_out, dim3((unsigned)ceil_div(N, 256)), dim3(256), 0, s, pidx, N,
                     logp_p, lse_p, logp, lse);
}

// ------------------------------------------------ Eq. 1 per-token term
// One thread per row. For a valid row of rollout b (weight c_b):
//   rho = exp(logp - old), pg = -min(rho*A, clip(rho)*A),
//   kl = exp(d) - d - 1 with d = ref - logp (evaluated as expm1(d) - d),
//   ell = pg + beta*kl, g = c_b*(dpg/dlogp + beta*(1 - exp(d))).
// Each block writes the sum of c_b*ell over its rows to loss_part.
__global__ void __launch_bounds__(256) k_token_objective(const TokenArgs a) {
  __shared__ float red[4];
  int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x;
  float contrib = 0.f;
  if (r < a.N) {
    int32_t j = a.pidx[r];
    float lp = 0.f, l = 0.f, ell = 0.f, g = 0.f;
    uint8_t clipped = 0;
    if (j >= 0 && a.objective == 1) {
      // cross-entropy: ell = -logp, dL/dlogp = -1/n_valid
      const float c = 1.f / (float)a.hdr->num_valid;
      lp = a.logp_p[j];
      l = a.lse_p[j];
      ell = -lp;
      g = -c;
      a.g_p[j] = g;
      contrib = c * ell;
    } else if (j >= 0) {
      int32_t b = a.seq_p[j];
      int32_t cnt = a.counts[b];
      float c = a.agg == 0 ? 1.f / ((float)a.B * (float)cnt) : 1.f / (float)a.hdr->num_valid;
      float A = a.adv[b];
      lp = a.logp_p[j];
      l = a.lse_p[j];
      float rho = __expf(lp - a.old_logp[r]);
      float rc = fminf(fmaxf(rho, 1.f - a.eps), 1.f + a.eps);
      float u = rho * A, cl = rc * A;
      float pg = -fminf(u, cl);
      float d = a.ref_logp ? a.ref_logp[r] - lp : 0.f;
      float em1 = expm1f(d);
      float kl = em1 - d;
      ell = pg + a.beta * kl;
      bool unclipped = u <= cl;
      float dpg = unclipped ? -A * rho : 0.f;
      g = c * (dpg - a.beta * em1);
      clipped = unclipped ? 0 : 1;
      a.g_p[j] = g;
      contrib = c * ell;
    }
    if (a.logp_out) a.logp_out[r] = lp;
    if (a.lse_out) a.lse_out[r] = l;
    if (a.token_loss) a.token_loss[r] = ell;
    if (a.dlogp) a.dlogp[r] = g;
    if (a.clip_flag) a.clip_flag[r] = clipped;
  }
  float t = block_sum_256(contrib, red);
  if (threadIdx.x == 0) a.loss_part[blockIdx.x] = t;
}

__global__ void __launch_bounds__(256) k_loss_final(const float* __restrict__ part, int64_t n,
                                                    float* __restrict__ loss) {
  __shared__ float red[4];
  float s = 0.f;
  for (int64_t i = threadIdx.x; i < n; i += 256) s += part[i];
  float t = block_sum_256(s, red);
  if (threadIdx.x == 0) *loss = t;
}

int64_t token_objective_blocks(int64_t N) { return ceil_div(N, 256); }

void launch_token_objective(const TokenArgs& a, hipStream_t s) {
  int64_t blocks = ceil_div(a.N, 256);
  hipLaunchKernelGGL(k_token_objective, dim3((unsigned)blocks), dim3(256), 0, s, a);
  hipLaunchKernelGGL(k_loss_final, dim3(1), dim3(256), 0, s, a.loss_part, blocks, a.loss);
}

// Zero the g of packed slots beyond the valid count (so padding contributes 0).
__global__ void __launch_bounds__(256) k_gather_dot_bf16(const uint16_t* __restrict__ hidden,
                                                         const uint16_t* __restrict__ W, int64_t H,
                                                         const int32_t* __restrict__ rows_p,
                                                         const int32_t* __restrict__ y_p,
                                                         const WsHeader* __restrict__ hdr,
                                                         float* __restrict__ zy) {
  int64_t j = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  int lane = threadIdx.x & 63;
  if (j >= hdr->num_valid) return;
  const uint16_t* h = hidden + (int64_t)rows_p[j] * H;
  const uint16_t* w = W + (int64_t)y_p[j] * H;
  float s = 0.f;
  for (int64_t k = lane * 8; k < H; k += 512) {
    u32x4 a = *(const u32x4*)(h + k), b = *(const u32x4*)(w + k);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      s = fmaf(__uint_as_float(a[q] << 16), __uint_as_float(b[q] << 16), s);
      s = fmaf(__uint_as_float(a[q] & 0xffff0000u), __uint_as_float(b[q] & 0xffff0000u), s);
    }
  }
  s = wave_sum(s);
  if (lane == 0) zy[j] = s;
}

void launch_gather_dot_bf16(const uint16_t* hidden, const uint16_t* W, int64_t H,
                            const int32_t* rows_p, const int32_t* y_p, const WsHeader* hdr,
                            float* zy, int64_t Nmax, hipStream_t s) {
  hipLaunchKernelGGL(k_gather_dot_bf16, dim3((unsigned)ceil_div(Nmax, 4)), dim3(256), 0, s, hidden,
                     W, H, rows_p, y_p, hdr, zy);
}

// ------------------------------------------------------- operand tiling
__global__ void __launch_bounds__(256) k_tile_rows(const uint16_t* __restrict__ in, int64_t ld_in,
                                                   const int32_t* __restrict__ rows,
                                                   int64_t n_static,
                                                   const WsHeader* __restrict__ hdr, int64_t K,
                                                   int64_t kb_per_row, int64_t stride,
                                                   uint16_t* __restrict__ out) {
  const int64_t rb = blockIdx.x / kb_per_row, kb = blockIdx.x - rb * kb_per_row;
  const int64_t blk = rb * stride + kb;
  const int64_t nvalid = hdr ? (int64_t)hdr->num_valid : n_static;
  const int t = threadIdx.x;
  const int64_t k0 = kb * 32 + (t & 3) * 8;
  uint16_t* ob = out + blk * kTileElems + (t & 3) * 8;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = (t >> 2) + 64 * i;
    const int64_t row = rb * 256 + r;
    u32x4 v = {0, 0, 0, 0};
    if (row < nvalid) {
      const uint16_t* p = in + (rows ? (int64_t)rows[row] : row) * ld_in + k0;
      if (k0 + 8 <= K) {
        v = *(const u32x4*)p;
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          uint32_t lo = k0 + 2 * q < K ? p[2 * q] : 0;
          uint32_t hi = k0 + 2 * q + 1 < K ? p[2 * q + 1] : 0;
          v[q] = lo | (hi << 16);
        }
      }
    }
    *(u32x4*)(ob + r * 32) = v;
  }
}

void launch_tile_rows(const uint16_t* in, int64_t ld_in, const int32_t* rows, int64_t n_static,
                      const WsHeader* hdr, int64_t r_pad, int64_t K, int64_t stride,
                      uint16_t* out, hipStream_t s) {
  const int64_t kb_per_row = ceil_div(K, 32);
  const int64_t blocks = r_pad / 256 * kb_per_row;
  hipLaunchKernelGGL(k_tile_rows, dim3((unsigned)blocks), dim3(256), 0, s, in, ld_in, rows,
                     n_static, hdr, K, kb_per_row, stride, out);
}

// n_pad must be a multiple of 64; `out` holds round_up(K, 256) x n_pad elements.
__global__ void __launch_bounds__(256) k_zero_masked_rows(const int32_t* __restrict__ pidx,
                                                          int64_t N, int64_t H, void* out,
                                                          int out_bf16) {
  int64_t r = blockIdx.x;
  if (r >= N || pidx[r] >= 0) return;
  if (out_bf16) {
    uint16_t* p = (uint16_t*)out + r * H;
    for (int64_t k = threadIdx.x; k < H; k += 256) p[k] = 0;
  } else {
    float* p = (float*)out + r * H;
    for (int64_t k = threadIdx.x; k < H; k += 256) p[k] = 0.f;
  }
}
void launch_zero_masked_rows(const int32_t* pidx, int64_t N, int64_t H, void* out, int out_bf16,
                             hipStream_t s) {
  hipLaunchKernelGGL(k_zero_masked_rows, dim3((unsigned)N), dim3(256), 0, s, pidx, N, H, out,
                     out_bf16);
}

// ------------------------------------------------------- AdamW step
// One pass over the parameters: each thread updates 4 consecutive elements
// (16-byte loads and stores of w, m, v, g; an 8-byte store of the bf16
// copy), grid-stride over the array; the last n % 4 elements are done one by
// one by the first threads.
__device__ __forceinline__ void adamw_one(float& w, float& m, float& v, float g,
                                          const AdamArgs& a) {
  m = a.beta1 * m + (1.f - a.beta1) * g;
  v = a.beta2 * v + (1.f - a.beta2) * g * g;
  const float denom = sqrtf(v) * a.inv_sqrt_bc2 + a.eps;
  w = w * a.decay - a.step_size * (m / denom);
}

__global__ void __launch_bounds__(256) k_adamw(AdamArgs a) {
  const int64_t n4 = a.n >> 2;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += stride) {
    f32x4 w = ((const f32x4*)a.w)[i];
    f32x4 m = ((const f32x4*)a.m)[i];
    f32x4 v = ((const f32x4*)a.v)[i];
    const f32x4 g = ((const f32x4*)a.g)[i];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float we = w[e], me = m[e], ve = v[e];
      adamw_one(we, me, ve, g[e], a);
      w[e] = we;
      m[e] = me;
      v[e] = ve;
    }
    ((f32x4*)a.w)[i] = w;
    ((f32x4*)a.m)[i] = m;
    ((f32x4*)a.v)[i] = v;
    if (a.w_bf16) {
      uint2 b = make_uint2(bf16_pack2(w[0], w[1]), bf16_pack2(w[2], w[3]));
      ((uint2*)a.w_bf16)[i] = b;
    }
  }
  const int64_t t = n4 * 4 + threadIdx.x;  // the last n % 4 elements
  if (blockIdx.x == 0 && t < a.n) {
    float w = a.w[t], m = a.m[t], v = a.v[t];
    adamw_one(w, m, v, a.g[t], a);
    a.w[t] = w;
    a.m[t] = m;
    a.v[t] = v;
    if (a.w_bf16) a.w_bf16[t] = bf16_bits(w);
  }
}

// ------------------------------------------------------------ split-K sum
__global__ void k_sum_splits(const float* __restrict__ part, int splits, int64_t stride,
                             int64_t ld_part, float* __restrict__ out, int64_t ld_out,
                             int64_t rows, int64_t cols, int accumulate) {
  const int64_t total = rows * cols;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / cols, c = i - r * cols;
    const float* p = part + r * ld_part + c;
    float acc = p[0];
    for (int sp = 1; sp < splits; ++sp) acc += p[sp * stride];
    out[r * ld_out + c] = accumulate ? out[r * ld_out + c] + acc : acc;
  }
}

void launch_sum_splits(const float* part, int splits, int64_t stride, int64_t ld_part, float* out,
                       int64_t ld_out, int64_t rows, int64_t cols, int accumulate, hipStream_t s) {
  const int64_t total = rows * cols;
  if (total <= 0) return;
  const int blocks = (int)(ceil_div(total, 256) < 16384 ? ceil_div(total, 256) : 16384);
  hipLaunchKernelGGL(k_sum_splits, dim3(blocks), dim3(256), 0, s, part, splits, stride, ld_part,
                     out, ld_out, rows, cols, accumulate);
}

// dL/dh rows from the K-split partials of the one dL/dh product: for packed
// row t < num_valid, the partials summed in split order, plus the sampled
// id's term g_t W[y_t] in fp32, rounded once into row rows_p[t] of the
// output. One workgroup per packed row, 4 columns per thread.
__global__ void __launch_bounds__(256) k_dh_finish(const float* __restrict__ part, int splits,
                                                   int64_t stride, int64_t ld,
                                                   const WsHeader* __restrict__ hdr, int64_t H,
                                                   const float* __restrict__ g_p,
                                                   const int32_t* __restrict__ y_p,
                                                   const uint16_t* __restrict__ W,
                                                   const int32_t* __restrict__ rows_p, void* out,
                                                   int out_bf16) {
  const int64_t t = blockIdx.x;
  if (t >= hdr->num_valid) return;
  const float g = g_p[t];
  const uint16_t* wr = W + (int64_t)y_p[t] * H;
  const int64_t orow = (int64_t)rows_p[t] * H;
  for (int64_t c = 4 * (int64_t)threadIdx.x; c < H; c += 4 * 256) {
    const float* p = part + t * ld + c;
    float v[4] = {p[0], p[1], p[2], p[3]};
    for (int sp = 1; sp < splits; ++sp)
      for (int k = 0; k < 4; ++k) v[k] += p[sp * stride + k];
    for (int k = 0; k < 4; ++k) v[k] += g * __uint_as_float((uint32_t)wr[c + k] << 16);
    if (out_bf16) {
      for (int k = 0; k < 4; ++k) ((uint16_t*)out)[orow + c + k] = bf16_bits(v[k]);
    } else {
      for (int k = 0; k < 4; ++k) ((float*)out)[orow + c + k] = v[k];
    }
  }
}

void launch_dh_finish(const float* part, int splits, int64_t stride, int64_t ld,
                      const WsHeader* hdr, int64_t rows, int64_t H, const float* g_p,
                      const int32_t* y_p, const uint16_t* W, const int32_t* rows_p, void* out,
                      int out_bf16, hipStream_t s) {
  if (rows <= 0) return;
  hipLaunchKernelGGL(k_dh_finish, dim3((unsigned)rows), dim3(256), 0, s, part, splits, stride, ld,
                     hdr, H, g_p, y_p, W, rows_p, out, out_bf16);
}

void launch_adamw(const AdamArgs& a, hipStream_t s) {
  const int64_t n4 = a.n >> 2;
  int64_t blocks = ceil_div(n4 > 0 ? n4 : 1, 256);
  if (blocks > 256 * 32) blocks = 256 * 32;  // 32 resident workgroups per CU, grid-stride beyond
  hipLaunchKernelGGL(k_adamw, dim3((unsigned)blocks), dim3(256), 0, s, a);
}

// ------------------------------------------------- plain fp32 path
// Scoring: one block per packed token; the hidden row sits in LDS and each
// thread walks a strided subset of the vocabulary with its own online
// (max, sum-exp), merged at the end in a fixed tree.
__global__ void __launch_bounds__(256) k_f32_score(const float* __restrict__ hidden,
                                                   const float* __restrict__ W, int64_t H,
                                                   int64_t V, const int32_t* __restrict__ rows_p,
                                                   const int32_t* __restrict__ y_p,
                                                   const WsHeader* __restrict__ hdr,
                                                   float* __restrict__ lse_p,
                                                   float* __restrict__ logp_p,
                                                   float* __restrict__ zy_p) {
  extern __shared__ float sh[];
  float* hs = sh;  // [H]
  __shared__ float rm[256], rs[256];
  __shared__ float zyv;
  int64_t j = blockIdx.x;
  if (j >= hdr->num_valid) return;
  const float* h = hidden + (int64_t)rows_p[j] * H;
  for (int64_t k = threadIdx.x; k < H; k += 256) hs[k] = h[k];
  __syncthreads();
  int32_t y = y_p[j];
  float m = -INFINITY, s = 0.f;
  for (int64_t v = threadIdx.x; v < V; v += 256) {
    const float* w = W + v * H;
    float z = 0.f;
    for (int64_t k = 0; k < H; ++k) z = fmaf(hs[k], w[k], z);
    if (v == y) zyv = z;
    lse_merge(m, s, z, 1.f);
  }
  rm[threadIdx.x] = m;
  rs[threadIdx.x] = s;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) {
      float mm = rm[threadIdx.x], ss = rs[threadIdx.x];
      lse_merge(mm, ss, rm[threadIdx.x + o], rs[threadIdx.x + o]);
      rm[threadIdx.x] = mm;
      rs[threadIdx.x] = ss;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    float l = rm[0] + logf(rs[0]);
    lse_p[j] = l;
    logp_p[j] = zyv - l;
    zy_p[j] = zyv;
  }
}

void launch_f32_score(const float* hidden, const float* W, int64_t H, int64_t V,
                      const int32_t* rows_p, const int32_t* y_p, const WsHeader* hdr,
                      float* lse_p, float* logp_p, float* zy_p, int64_t Nmax, hipStream_t s) {
  hipLaunchKernelGGL(k_f32_score, dim3((unsigned)Nmax), dim3(256), (size_t)H * 4, s, hidden, W, H,
                     V, rows_p, y_p, hdr, lse_p, logp_p, zy_p);
}

// dL/dh for one packed token per block: walks the vocabulary in slabs of 256
// rows, recomputing z and dz = g*(1[v=y] - exp(z - lse)), and accumulates
// sum_v dz_v W_v into an LDS row.
__global__ void __launch_bounds__(256) k_f32_grad_hidden(const float* __restrict__ hidden,
                                                         const float* __restrict__ W, int64_t H,
                                                         int64_t V,
                                                         const int32_t* __restrict__ rows_p,
                                                         const int32_t* __restrict__ y_p,
                                                         const float* __restrict__ lse_p,
                                                         const float* __restrict__ g_p,
                                                         const WsHeader* __restrict__ hdr,
                                                         float* __restrict__ grad_hidden) {
  extern __shared__ float sh[];
  float* hs = sh;       // [H]
  float* acc = sh + H;  // [H]
  __shared__ float dzs[256];
  int64_t j = blockIdx.x;
  if (j >= hdr->num_valid) return;
  int64_t row = rows_p[j];
  const float* h = hidden + row * H;
  for (int64_t k = threadIdx.x; k < H; k += 256) {
    hs[k] = h[k];
    acc[k] = 0.f;
  }
  __syncthreads();
  float g = g_p[j], l = lse_p[j];
  int32_t y = y_p[j];
  for (int64_t v0 = 0; v0 < V; v0 += 256) {
    int64_t v = v0 + threadIdx.x;
    float dz = 0.f;
    if (v < V && g != 0.f) {
      const float* w = W + v * H;
      float z = 0.f;
      for (int64_t k = 0; k < H; ++k) z = fmaf(hs[k], w[k], z);
      dz = g * ((v == y ? 1.f : 0.f) - __expf(z - l));
    }
    dzs[threadIdx.x] = dz;
    __syncthreads();
    int64_t vn = V - v0 < 256 ? V - v0 : 256;
    for (int64_t k = threadIdx.x; k < H; k += 256) {
      float a = acc[k];
      for (int64_t q = 0; q < vn; ++q) a = fmaf(dzs[q], W[(v0 + q) * H + k], a);
      acc[k] = a;
    }
    __syncthreads();
  }
  float* out = grad_hidden + row * H;
  for (int64_t k = threadIdx.x; k < H; k += 256) out[k] = acc[k];
}

void launch_f32_grad_hidden(const float* hidden, const float* W, int64_t H, int64_t V,
                            const int32_t* rows_p, const int32_t* y_p, const float* lse_p,
                            const float* g_p, const WsHeader* hdr, float* grad_hidden,
                            int64_t Nmax, hipStream_t s) {
  hipLaunchKernelGGL(k_f32_grad_hidden, dim3((unsigned)Nmax), dim3(256), (size_t)H * 8, s, hidden,
                     W, H, V, rows_p, y_p, lse_p, g_p, hdr, grad_hidden);
}

// dL/dW for one vocabulary row per block: walks the packed tokens in slabs
// of 256, recomputing z and dz, and accumulates sum_t dz_t h_t.
__global__ void __launch_bounds__(256) k_f32_grad_weight(const float* __restrict__ hidden,
                                                         const float* __restrict__ W, int64_t H,
                                                         int64_t V,
                                                         const int32_t* __restrict__ rows_p,
                                                         const int32_t* __restrict__ y_p,
                                                         const float* __restrict__ lse_p,
                                                         const float* __restrict__ g_p,
                                                         const WsHeader* __restrict__ hdr,
                                                         float* __restrict__ grad_weight,
                                                         int accumulate) {
  extern __shared__ float sh[];
  float* ws = sh;       // [H]
  float* acc = sh + H;  // [H]
  __shared__ float dzs[256];
  __shared__ int32_t rws[256];
  int64_t v = blockIdx.x;
  const float* w = W + v * H;
  for (int64_t k = threadIdx.x; k < H; k += 256) {
    ws[k] = w[k];
    acc[k] = 0.f;
  }
  __syncthreads();
  int64_t n = hdr->num_valid;
  for (int64_t t0 = 0; t0 < n; t0 += 256) {
    int64_t j = t0 + threadIdx.x;
    float dz = 0.f;
    int32_t row = 0;
    if (j < n) {
      row = rows_p[j];
      float g = g_p[j];
      if (g != 0.f) {
        const float* h = hidden + (int64_t)row * H;
        float z = 0.f;
        for (int64_t k = 0; k < H; ++k) z = fmaf(h[k], ws[k], z);
        dz = g * ((v == y_p[j] ? 1.f : 0.f) - __expf(z - lse_p[j]));
      }
    }
    dzs[threadIdx.x] = dz;
    rws[threadIdx.x] = row;
    __syncthreads();
    int64_t tn = n - t0 < 256 ? n - t0 : 256;
    for (int64_t k = threadIdx.x; k < H; k += 256) {
      float a = acc[k];
      for (int64_t q = 0; q < tn; ++q) a = fmaf(dzs[q], hidden[(int64_t)rws[q] * H + k], a);
      acc[k] = a;
    }
    __syncthreads();
  }
  float* out = grad_weight + v * H;
  for (int64_t k = threadIdx.x; k < H; k += 256) out[k] = accumulate ? out[k] + acc[k] : acc[k];
}

void launch_f32_grad_weight(const float* hidden, const float* W, int64_t H, int64_t V,
                            const int32_t* rows_p, const int32_t* y_p, const float* lse_p,
                            const float* g_p, const WsHeader* hdr, float* grad_weight,
                            int accumulate, hipStream_t s) {
  hipLaunchKernelGGL(k_f32_grad_weight, dim3((unsigned)V), dim3(256), (size_t)H * 8, s, hidden, W,
                     H, V, rows_p, y_p, lse_p, g_p, hdr, grad_weight, accumulate);
}

}  // namespace grpo
