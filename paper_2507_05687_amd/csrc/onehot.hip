// The sampled id's term of dL/dW, applied exactly in fp32.
//
// dz_{t,v} = g_t (1[v = y_t] - p_{t,v}) (Sec. 3.3, Eq. 1, differentiated
// through the log-softmax). The bf16 dz operand of the MFMA products carries
// only -g_t p_{t,v}; its largest entry, g_t at v = y_t, would otherwise be
// rounded to bf16 and dominate the gradients' error. dL/dh gets g_t W_{y_t}
// in the product's epilogue; dL/dW gets, for every id v,
//
//   sum over the valid tokens t with y_t = v of g_t h_t,
//
// here. The tokens are grouped by id with a stable LSD radix sort (8-bit
// digits) of the packed ids, so that each id's sum runs over its tokens in
// packed order: the result is the same bits on every run. No kernel uses
// atomics; digit ranks within a wave come from ballots.
#include "kernels.h"

namespace grpo {

constexpr int kSortTile = 4096;  // items per workgroup of the radix passes (256 threads x 16)

// keys[i] = id of packed row i for the valid rows, `sentinel` (above every
// id) for the rest; vals[i] = i
__global__ void __launch_bounds__(256) k_sort_init(const int32_t* __restrict__ y_p,
                                                   const WsHeader* __restrict__ hdr, int64_t n,
                                                   int32_t sentinel, int32_t* __restrict__ keys,
                                                   int32_t* __restrict__ vals) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  keys[i] = i < hdr->num_valid ? y_p[i] : sentinel;
  vals[i] = (int32_t)i;
}

// Lanes of this wave whose digit equals this lane's (among lanes with `valid`).
__device__ __forceinline__ uint64_t match_digit(int d, bool valid) {
  uint64_t m = __ballot(valid);
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const uint64_t bal = __ballot((d >> b) & 1);
    m &= ((d >> b) & 1) ? bal : ~bal;
  }
  return valid ? m : 0;
}

// counts[d * tiles + tile] = items of the tile whose digit (key >> shift) & 255 is d
__global__ void __launch_bounds__(256) k_radix_count(const int32_t* __restrict__ keys, int64_t n,
                                                     int shift, int64_t tiles,
                                                     int32_t* __restrict__ counts) {
  __shared__ int32_t cnt[4][256];
  const int t = threadIdx.x, w = t >> 6, lane = t & 63;
  for (int k = t; k < 1024; k += 256) (&cnt[0][0])[k] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * kSortTile;
  for (int r = 0; r < kSortTile / 256; ++r) {
    const int64_t i = base + r * 256 + t;
    const bool valid = i < n;
    const int d = valid ? (keys[i] >> shift) & 255 : 0;
    const uint64_t m = match_digit(d, valid);
    // the group's highest lane adds the group's size (one writer per digit and wave)
    if (valid && (m >> lane) == 1ull) cnt[w][d] += __popcll(m);
  }
  __syncthreads();
  counts[(int64_t)t * tiles + blockIdx.x] = (cnt[0][t] + cnt[1][t]) + (cnt[2][t] + cnt[3][t]);
}

// exclusive prefix sum of counts[0..total) in place (one workgroup)
__global__ void __launch_bounds__(1024) k_radix_scan(int32_t* __restrict__ counts, int64_t total) {
  __shared__ int32_t part[1024];
  const int t = threadIdx.x;
  const int64_t per = (total + 1023) / 1024;
  const int64_t b = t * per, e = b + per < total ? b + per : total;
  int32_t s = 0;
  for (int64_t i = b; i < e; ++i) s += counts[i];
  part[t] = s;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {  // inclusive scan of the per-thread sums
    const int32_t v = t >= o ? part[t - o] : 0;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  int32_t run = t > 0 ? part[t - 1] : 0;
  for (int64_t i = b; i < e; ++i) {
    const int32_t c = counts[i];
    counts[i] = run;
    run += c;
  }
}

// stable scatter by digit: the tile's items keep their order within a digit
__global__ void __launch_bounds__(256) k_radix_scatter(const int32_t* __restrict__ keys,
                                                       const int32_t* __restrict__ vals, int64_t n,
                                                       int shift, int64_t tiles,
                                                       const int32_t* __restrict__ offsets,
                                                       int32_t* __restrict__ keys_out,
                                                       int32_t* __restrict__ vals_out) {
  __shared__ int32_t run[256];
  __shared__ int32_t wc[4][256];
  const int t = threadIdx.x, w = t >> 6, lane = t & 63;
  run[t] = offsets[(int64_t)t * tiles + blockIdx.x];
  for (int k = t; k < 1024; k += 256) (&wc[0][0])[k] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * kSortTile;
  const uint64_t below = (1ull << lane) - 1;
  for (int r = 0; r < kSortTile / 256; ++r) {
    const int64_t i = base + r * 256 + t;
    const bool valid = i < n;
    const int32_t key = valid ? keys[i] : 0;
    const int32_t val = valid ? vals[i] : 0;
    const int d = (key >> shift) & 255;
    const uint64_t m = match_digit(d, valid);
    if (valid && (m >> lane) == 1ull) wc[w][d] = __popcll(m);
    __syncthreads();
    if (valid) {
      int32_t pos = run[d] + __popcll(m & below);
      for (int v = 0; v < w; ++v) pos += wc[v][d];
      keys_out[pos] = key;
      vals_out[pos] = val;
    }
    __syncthreads();
    run[t] += (wc[0][t] + wc[1][t]) + (wc[2][t] + wc[3][t]);
    wc[0][t] = wc[1][t] = wc[2][t] = wc[3][t] = 0;
    __syncthreads();
  }
}

// One wave per sorted position; the first position of each id's run adds
// sum_t g_t h_t over the run (packed order) to that id's dL/dW row. A lane
// covers 8 consecutive columns; columns are walked 512 at a time.
__global__ void __launch_bounds__(256) k_onehot_dw(const int32_t* __restrict__ keys,
                                                   const int32_t* __restrict__ perm,
                                                   const WsHeader* __restrict__ hdr,
                                                   const int32_t* __restrict__ rows_p,
                                                   const float* __restrict__ g_p,
                                                   const uint16_t* __restrict__ hidden, int64_t H,
                                                   float* __restrict__ dW) {
  const int64_t k = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int64_t nv = hdr->num_valid;
  if (k >= nv) return;
  const int32_t y = keys[k];
  if (k > 0 && keys[k - 1] == y) return;
  int64_t e = k + 1;
  while (e < nv && keys[e] == y) ++e;
  float* row = dW + (int64_t)y * H;
  for (int64_t c0 = (int64_t)lane * 8; c0 < H; c0 += 512) {
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int64_t q = k; q < e; ++q) {
      const int32_t p = perm[q];
      const float g = g_p[p];
      const u32x4 v = *(const u32x4*)(hidden + (int64_t)rows_p[p] * H + c0);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        acc[2 * j] += g * __uint_as_float(v[j] << 16);
        acc[2 * j + 1] += g * __uint_as_float(v[j] & 0xffff0000u);
      }
    }
    float prev[8];  // dL/dW needs only 4-byte alignment: scalar accesses
#pragma unroll
    for (int j = 0; j < 8; ++j) prev[j] = row[c0 + j];
#pragma unroll
    for (int j = 0; j < 8; ++j) row[c0 + j] = prev[j] + acc[j];
  }
}

int onehot_sort_passes(int64_t V) {
  int bits = 1;
  while ((1ll << bits) <= V) ++bits;  // the sentinel 2^bits - 1 lies above every id
  return (bits + 7) / 8;
}

int64_t onehot_count_entries(int64_t n) { return 256 * ceil_div(n, kSortTile); }

void launch_onehot_dw(const OnehotArgs& a, hipStream_t s) {
  const int passes = onehot_sort_passes(a.V);
  const int32_t sentinel = (int32_t)((1ll << (8 * passes < 31 ? 8 * passes : 31)) - 1);
  const int64_t tiles = ceil_div(a.n, kSortTile);
  hipLaunchKernelGGL(k_sort_init, dim3((unsigned)ceil_div(a.n, 256)), dim3(256), 0, s, a.y_p,
                     a.hdr, a.n, sentinel, a.keys[0], a.vals[0]);
  for (int p = 0; p < passes; ++p) {
    const int in = p & 1;
    hipLaunchKernelGGL(k_radix_count, dim3((unsigned)tiles), dim3(256), 0, s, a.keys[in], a.n,
                       8 * p, tiles, a.counts);
    hipLaunchKernelGGL(k_radix_scan, dim3(1), dim3(1024), 0, s, a.counts, 256 * tiles);
    hipLaunchKernelGGL(k_radix_scatter, dim3((unsigned)tiles), dim3(256), 0, s, a.keys[in],
                       a.vals[in], a.n, 8 * p, tiles, a.counts, a.keys[in ^ 1], a.vals[in ^ 1]);
  }
  const int out = passes & 1;
  hipLaunchKernelGGL(k_onehot_dw, dim3((unsigned)ceil_div(a.n, 4)), dim3(256), 0, s, a.keys[out],
                     a.vals[out], a.hdr, a.rows_p, a.g_p, a.hidden, a.H, a.dW);
}

}  // namespace grpo
