// Host side of libgrpo: argument validation, workspace layout, the launch
// sequence of each entry point, and optional per-kernel event timing.
// Declarations and argument contracts are in include/grpo.h.
#include "grpo.h"

#include <math.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <vector>

#include "kernels.h"

using namespace grpo;

namespace {

// --------------------------------------------------------- kernel timing
enum Kind {
  K_PACK, K_ADV, K_GEMM_LSE, K_LSE_FIN, K_TOKEN, K_GEMM_DZ, K_GEMM_DH, K_GEMM_DW,
  K_F32_SCORE, K_F32_DH, K_F32_DW, K_ZERO_ROWS, K_GATHER_DOT, K_TILE, K_ADAMW,
  K_RULE_REWARD, K_SUM_SPLITS, K_ONEHOT, K_DH_FINISH, K_NUM_KINDS
};
const char* kKindNames[K_NUM_KINDS] = {
    "pack_valid",  "group_advantages", "gemm_logits_lse", "lse_finalize",   "token_objective",
    "gemm_recompute_dz", "gemm_grad_hidden", "gemm_grad_weight", "f32_score",
    "f32_grad_hidden", "f32_grad_weight", "zero_masked_rows", "gather_dot", "tile", "adamw",
    "rule_reward", "sum_splits", "onehot_grad_weight", "dh_finish"};

struct Prof {
  std::mutex mu;
  bool on = false;
  struct Rec { int kind; hipEvent_t a, b; };
  std::vector<Rec> recs;
  int64_t launches[K_NUM_KINDS] = {};
  double ms[K_NUM_KINDS] = {};
};
Prof& prof() {
  static Prof p;
  return p;
}

// Folds finished event pairs into the per-kind totals (waits for them).
// Caller holds p.mu.
grpo_status fold_records(Prof& p) {
  for (auto& r : p.recs) {
    if (hipEventSynchronize(r.b) != hipSuccess) return GRPO_ERR_HIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return GRPO_ERR_HIP;
    p.launches[r.kind] += 1;
    p.ms[r.kind] += ms;
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  p.recs.clear();
  return GRPO_OK;
}
constexpr size_t kMaxPendingRecords = 4096;  // event pairs held before they are folded

// Runs `launch` bracketed by events when timing is on. A launch failure is
// told apart from an error the calling thread had already left pending: the
// last-error state is only peeked at, and consumed only when it is ours.
template <class F>
grpo_status timed(int kind, hipStream_t s, F&& launch) {
  Prof& p = prof();
  bool on;
  {
    std::lock_guard<std::mutex> g(p.mu);
    on = p.on;
  }
  hipEvent_t a = nullptr, b = nullptr;
  if (on) {
    if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) return GRPO_ERR_HIP;
    if (hipEventRecord(a, s) != hipSuccess) return GRPO_ERR_HIP;
  }
  const hipError_t before = hipPeekAtLastError();
  launch();
  if (before == hipSuccess && hipPeekAtLastError() != hipSuccess) {
    (void)hipGetLastError();
    return GRPO_ERR_HIP;
  }
  if (on) {
    if (hipEventRecord(b, s) != hipSuccess) return GRPO_ERR_HIP;
    std::lock_guard<std::mutex> g(p.mu);
    p.recs.push_back({kind, a, b});
    if (p.recs.size() >= kMaxPendingRecords) return fold_records(p);
  }
  return GRPO_OK;
}

#define TRY(x)                          \
  do {                                  \
    grpo_status st_ = (x);              \
    if (st_ != GRPO_OK) return st_;     \
  } while (0)

// --------------------------------------------------------- device check
grpo_status check_device() {
  static std::mutex mu;
  static int checked[64] = {};  // 0 unknown, 1 ok, 2 bad
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return GRPO_ERR_DEVICE;
  std::lock_guard<std::mutex> g(mu);
  if (checked[dev] == 0) {
    hipDeviceProp_t p;
    if (hipGetDeviceProperties(&p, dev) != hipSuccess) return GRPO_ERR_DEVICE;
    checked[dev] = strncmp(p.gcnArchName, "gfx950", 6) == 0 ? 1 : 2;
  }
  return checked[dev] == 1 ? GRPO_OK : GRPO_ERR_DEVICE;
}

// --------------------------------------------------------- static scratch
// grpo_pack_valid_static's scratch: the workspace header (error words and the
// valid count) and the per-rollout offsets, in a file-scope device array that
// every GPU the library runs on holds until the process ends. Host code uses
// the array only through the device address hipGetSymbolAddress returns for
// the current device (kept per device); the array's name is not a device
// address in host code.
constexpr int64_t kStaticMaxSeqs = 1 << 20;  // rollouts per call
constexpr size_t kStaticScratchBytes = 256 + 4 * ((size_t)kStaticMaxSeqs + 64);
static __device__ __align__(256) char scratch[kStaticScratchBytes];

grpo_status static_scratch(char** out) {
  static std::mutex mu;
  static char* addr[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return GRPO_ERR_DEVICE;
  std::lock_guard<std::mutex> g(mu);
  if (addr[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr)
      return GRPO_ERR_HIP;
    addr[dev] = (char*)ptr;
  }
  *out = addr[dev];
  return GRPO_OK;
}

// --------------------------------------------------------- workspace
constexpr size_t kAlign = 256;
constexpr int64_t kPackSeg = 4096;  // rows per packing workgroup without cu_seqlens
constexpr int64_t kMaxAdvPrompts = 4 * ((1ll << 24) - 1);  // group_advantages' grid limit
constexpr size_t kDefaultDzBudget = (size_t)16 << 30;  // bytes for the bf16 dz chunks
constexpr int64_t kVcMax = 8192;                        // columns per vocabulary chunk
constexpr int64_t kScoreRows = 8192;  // vocabulary rows per scoring launch (a multiple of 256)

struct Layout {
  int64_t Npad = 0, Vpad = 0, tiles_v = 0, Vc = 0, nchunks = 0, dh_group = 0;
  int dw_splits_max = 1;  // the most K splits of a dL/dW product (its partials' room)
  int dh_splits = 1;      // K splits of the dL/dh product when there is only one
  int64_t R = 0;  // rows of the token-indexed tiled buffers: the valid-row capacity, padded
  size_t hdr = 0, rows = 0, seq = 0, y = 0, pidx = 0, counts = 0, base = 0;
  size_t lse = 0, zy = 0, logp = 0, g = 0, ms = 0, lpart = 0;
  int64_t Hk = 0;  // H rounded up to the tiled block width
  // tiled buffers and their tile-row strides in blocks
  size_t WK = 0, hK = 0, dz = 0, dhacc = 0, dwpart = 0, dhpart = 0;
  const uint16_t* WKx = nullptr;  // the caller's tiled weight (no WK in the workspace)
  size_t okeys[2] = {0, 0}, ovals[2] = {0, 0}, ocounts = 0;  // sort of the sampled ids
  int64_t sK = 0, sChunk = 0;
  size_t total = 0;
};

// Tile-rows of a tiled buffer are one block further apart than their length,
// so that the blocks that concurrent tiles read at the same K step do not
// all share the same low address bits (and L2 sets).
int64_t tile_stride(int64_t K) { return ceil_div(K, kBK) + 1; }

// K splits for a product of `tiles` output tiles: the count up to kMaxSplits
// that best fills whole rounds of 256 workgroups (one per CU), taking more
// splits only for at least 2% more fill (each adds a pass over fp32
// partials). 512 tiles stay whole; 336 (a 5376-row chunk at H = 4096) take 3.
constexpr int kMaxSplits = 8;
int fill_splits(int64_t tiles) {
  if (tiles <= 0) return 1;
  int best = 1;
  double best_fill = 0;
  for (int sp = 1; sp <= kMaxSplits; ++sp) {
    const int64_t wg = sp * tiles;
    const double fill = (double)wg / (double)(256 * ceil_div(wg, 256));
    if (fill > best_fill + (sp == 1 ? 0.0 : 0.02)) {
      best = sp;
      best_fill = fill;
    }
  }
  return best;
}

size_t take(size_t& cur, size_t bytes) {
  size_t at = cur;
  cur += (bytes + kAlign - 1) / kAlign * kAlign;
  return at;
}

// Estimated seconds of the parts of the backward pass that depend on the
// vocabulary chunking: the dL/dW products (whole rounds of 256 workgroups,
// each a 256 x 256 tile over K = R tokens at about 1.9 PFLOP/s), the fp32
// partials of a split K (written and read once), the passes over the fp32
// dL/dh accumulator (read and written by every dL/dh product after the
// first) at about 5 TB/s, and a few launches per chunk.
double chunking_cost(int64_t R, int64_t Vpad, int64_t Hpad, int64_t Vc, int64_t group) {
  const double kFlops = 1.9e15, kBytes = 5e12, kLaunch = 20e-6;
  const double t_round = 256.0 * 2 * kTile * kTile * (double)R / kFlops;
  const int64_t n = ceil_div(Vpad, Vc);
  double t = 0;
  for (int c = 0; c < 2; ++c) {  // the n - 1 full chunks, then the last
    const int64_t cols = c == 0 ? Vc : Vpad - (n - 1) * Vc;
    const int64_t cnt = c == 0 ? n - 1 : 1;
    const int64_t tiles = cols / kTile * (Hpad / kTile);
    const int sp = fill_splits(tiles);
    double tc = (double)ceil_div(sp * tiles, 256) / sp * t_round + 3 * kLaunch;
    if (sp > 1) tc += 2.0 * sp * (double)cols * Hpad * 4 / kBytes;
    t += cnt * tc;
  }
  t += (ceil_div(n, group) - 1) * 8.0 * (double)R * Hpad / kBytes;
  return t;
}

// Vocabulary chunks of the backward pass and how many of them one dL/dh
// product takes. The token-major bf16 dz buffer holds `group` chunks of Vc
// columns for R rows and stays within `budget` bytes (0: kDefaultDzBudget):
// a small batch may hold the whole vocabulary (one dL/dh product, no
// accumulator). Vc (a multiple of 256, at most kVcMax) and the group are the pair
// of least chunking_cost; all chunks but the last are Vc wide.
void chunking(int64_t R, int64_t Vpad, int64_t Hpad, size_t budget, int64_t& Vc,
              int64_t& nchunks, int64_t& group) {
  if (budget == 0) budget = kDefaultDzBudget;
  int64_t cols = (int64_t)(budget / (2 * (size_t)R)) / kTile * kTile;
  if (cols > Vpad) cols = Vpad;
  if (cols < kTile) cols = kTile;
  int64_t cap = cols < kVcMax ? cols : kVcMax;
  if (cap > Vpad) cap = Vpad;
  double best = 0;
  for (int64_t c = cap; c >= kTile; c -= kTile) {
    const int64_t n = ceil_div(Vpad, c);
    int64_t gr = cols >= Vpad ? n : cols / c;  // the whole vocabulary: one group
    if (gr > n) gr = n;
    const double cost = chunking_cost(R, Vpad, Hpad, c, gr);
    if (c == cap || cost < best * 0.999) {
      best = cost;
      Vc = c;
      group = gr;
    }
  }
  nchunks = ceil_div(Vpad, Vc);
}

// max_valid: the most valid rows a call will have (0: all N); dz_budget: bytes
// for the logits-gradient chunks (0: the default).
Layout layout(grpo_op op, grpo_dtype dt, int64_t N, int64_t H, int64_t V, int64_t B,
              int64_t max_valid, size_t dz_budget, bool tiled_weight = false) {
  Layout L;
  L.Npad = round_up(N, kTile);
  L.Vpad = round_up(V, kTile);
  L.tiles_v = L.Vpad / kTile;
  L.R = round_up(max_valid > 0 && max_valid < N ? max_valid : N, kTile);
  size_t c = 0;
  L.hdr = take(c, sizeof(WsHeader));
  L.rows = take(c, 4 * L.Npad);
  L.seq = take(c, 4 * L.Npad);
  L.y = take(c, 4 * L.Npad);
  L.pidx = take(c, 4 * N);
  // per rollout, or per packing segment when every row forms one rollout
  const int64_t units = B > ceil_div(N, kPackSeg) ? B : ceil_div(N, kPackSeg);
  L.counts = take(c, 4 * units);
  L.base = take(c, 4 * (units + 1));
  L.lse = take(c, 4 * L.Npad);
  L.zy = take(c, 4 * L.Npad);
  L.logp = take(c, 4 * L.Npad);
  L.g = take(c, 4 * L.Npad);
  L.lpart = take(c, 4 * token_objective_blocks(N));
  if (dt == GRPO_BF16) {
    L.ms = take(c, 8 * L.tiles_v * L.R);  // one (max, sum-exp) partial per vocabulary tile
    // tiled copies of W and of the valid hidden rows (K = H contiguous blocks)
    L.Hk = round_up(H, kBK);
    L.sK = tile_stride(H);
    if (!tiled_weight) L.WK = take(c, 2 * L.Vpad * L.sK * kBK);
    L.hK = take(c, 2 * L.R * L.sK * kBK);
    if (op == GRPO_OP_LOSS_FWD_BWD) {
      const int64_t Hpad = round_up(H, kTile);
      chunking(L.R, L.Vpad, Hpad, dz_budget, L.Vc, L.nchunks, L.dh_group);
      // the group buffer: dh_group chunks, or the padded vocabulary when one
      // group holds every chunk (the last one narrower)
      L.sChunk = tile_stride(L.dh_group == L.nchunks ? L.Vpad : L.dh_group * L.Vc);
      L.dz = take(c, 2 * L.R * L.sChunk * kBK);
      // fp32 dh accumulator with every row and column of every tile present
      if (L.nchunks > L.dh_group) L.dhacc = take(c, 4 * L.R * Hpad);
      // dW partials of a split K (chunks too narrow to fill the GPU)
      const int64_t last = L.Vpad - (L.nchunks - 1) * L.Vc;
      const int sp_full = fill_splits(L.Vc / kTile * (Hpad / kTile));
      const int sp_last = fill_splits(last / kTile * (Hpad / kTile));
      L.dw_splits_max = sp_full > sp_last ? sp_full : sp_last;
      if (L.dw_splits_max > 1) L.dwpart = take(c, 4 * L.dw_splits_max * L.Vc * Hpad);
      // a single dL/dh product over few row tiles: a split K fills the GPU
      // (fp32 partials, summed with the sampled id's term by k_dh_finish)
      if (L.dh_group == L.nchunks) {
        L.dh_splits = fill_splits(L.R / kTile * (Hpad / kTile));
        if (L.dh_splits > 1) L.dhpart = take(c, 4 * (size_t)L.dh_splits * L.R * Hpad);
      }
      // the stable sort of the packed ids for the sampled-id term of dL/dW
      for (int b = 0; b < 2; ++b) {
        L.okeys[b] = take(c, 4 * L.R);
        L.ovals[b] = take(c, 4 * L.R);
      }
      L.ocounts = take(c, 4 * onehot_count_entries(L.R));
    }
  }
  L.total = c;
  return L;
}

template <class T>
T* at(void* ws, size_t off) {
  return (T*)((char*)ws + off);
}

// The tiled weight the products read: the caller's, else the workspace copy.
const uint16_t* weight_k(const Layout& L, void* ws) {
  return L.WKx ? L.WKx : at<uint16_t>(ws, L.WK);
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

grpo_status check_sizes(grpo_dtype dt, int64_t N, int64_t H, int64_t V) {
  if (dt != GRPO_F32 && dt != GRPO_BF16) return GRPO_ERR_DTYPE;
  if (N < 1 || H < 1 || V < 1) return GRPO_ERR_SHAPE;
  if (N >= (1ll << 31) - kTile || V >= (1ll << 31) - kTile || H >= (1ll << 20)) return GRPO_ERR_SHAPE;
  if (dt == GRPO_BF16 && H % 8 != 0) return GRPO_ERR_SHAPE;
  if (dt == GRPO_F32 && H > 8192) return GRPO_ERR_SHAPE;  // two LDS rows of H floats
  // the scoring product's grid (whole bands of 32 tile-rows) counts in 32 bits
  if (dt == GRPO_BF16 && (ceil_div(V, kTile) + 32) * ceil_div(N, kTile) >= (1ll << 31))
    return GRPO_ERR_SHAPE;
  return GRPO_OK;
}

// The bf16 backward: dL/dW contracts over the tokens, and the MFMA loop
// addresses its K steps (16 KiB each) with a 32-bit offset.
constexpr int64_t kMaxBwdTokens = 1ll << 22;
grpo_status check_bwd_sizes(grpo_dtype dt, int64_t N, int64_t H, int64_t V) {
  TRY(check_sizes(dt, N, H, V));
  return dt == GRPO_BF16 && N > kMaxBwdTokens ? GRPO_ERR_SHAPE : GRPO_OK;
}

// weight_tiled: bf16 only, 256-byte aligned (the layout of grpo_tile_weight)
grpo_status check_weight_tiled(grpo_dtype dt, const void* weight_tiled) {
  if (!weight_tiled) return GRPO_OK;
  if (dt != GRPO_BF16) return GRPO_ERR_DTYPE;
  return aligned(weight_tiled, kAlign) ? GRPO_OK : GRPO_ERR_ALIGN;
}

grpo_status check_ws(void* ws, size_t bytes, const Layout& L) {
  if (ws == nullptr) return GRPO_ERR_WORKSPACE;
  if (!aligned(ws, kAlign)) return GRPO_ERR_WORKSPACE;
  if (bytes < L.total) return GRPO_ERR_WORKSPACE;
  return GRPO_OK;
}

// Operands in the tiled layout: A has a_kt blocks per tile-row, B b_kt.
GemmArgs gemm_args(const void* A, int64_t a_kt, int64_t M, const void* B, int64_t b_kt,
                   int64_t N, const int32_t* m_dev, const int32_t* n_dev, int64_t K,
                   const int32_t* k_dev) {
  GemmArgs g;
  g.A = (const uint16_t*)A;
  g.M = (int)M;
  g.B = (const uint16_t*)B;
  g.N = (int)N;
  g.m_dev = m_dev;
  g.n_dev = n_dev;
  g.a_kt = a_kt;
  g.b_kt = b_kt;
  g.a_kb0 = g.b_kb0 = 0;
  g.a_cb0 = g.b_cb0 = 0;
  g.K = (int)K;
  g.k_dev = k_dev;
  g.tiles_m = (int)ceil_div(M, kTile);
  g.tiles_n = (int)ceil_div(N, kTile);
  g.splits = 1;
  return g;
}

// Packing shared by every entry point that takes a mask.
grpo_status run_pack(const Layout& L, void* ws, const uint8_t* mask, const int64_t* tokens,
                     int64_t V, const int64_t* cu, int64_t B, int64_t N, int32_t* rows_out,
                     int32_t* counts_out, int32_t* nvalid_out, hipStream_t s) {
  // the valid rows the workspace's token buffers hold (all N for the fp32 path)
  const int64_t cap = L.hK ? L.R : N;
  PackArgs a;
  a.mask = mask;
  a.tokens = tokens;
  a.V = V;
  a.cu = cu;
  // without cu_seqlens every row belongs to one rollout; it is packed in
  // segments, one workgroup each (the per-row rollout index is then unused)
  a.seg = kPackSeg;
  a.B = cu ? B : ceil_div(N, kPackSeg);
  a.N = N;
  a.counts = counts_out ? counts_out : at<int32_t>(ws, L.counts);
  a.base = at<int32_t>(ws, L.base);
  a.rows_p = rows_out ? rows_out : at<int32_t>(ws, L.rows);
  a.seq_p = at<int32_t>(ws, L.seq);
  a.y_p = tokens ? at<int32_t>(ws, L.y) : nullptr;
  a.pidx = at<int32_t>(ws, L.pidx);
  a.num_valid_out = nvalid_out;
  a.cap = cap;
  a.hdr = at<WsHeader>(ws, L.hdr);
  return timed(K_PACK, s, [&] { launch_pack(a, s); });
}

// Tiled copies of W (all V rows; not when the caller gave a tiled W) and of
// the valid hidden rows in packed order, the operands of the scoring and dz
// products.
grpo_status run_tiles(const Layout& L, void* ws, const void* hidden, const void* weight,
                      int64_t H, int64_t V, hipStream_t s) {
  const int32_t* rows_p = at<int32_t>(ws, L.rows);
  const WsHeader* hdr = at<WsHeader>(ws, L.hdr);
  if (!L.WKx) {
    TRY(timed(K_TILE, s, [&] {
      launch_tile_rows((const uint16_t*)weight, H, nullptr, V, nullptr, L.Vpad, H, L.sK,
                       at<uint16_t>(ws, L.WK), s);
    }));
  }
  return timed(K_TILE, s, [&] {
    launch_tile_rows((const uint16_t*)hidden, H, rows_p, 0, hdr, L.R, H, L.sK,
                     at<uint16_t>(ws, L.hK), s);
  });
}

// Forward vocabulary pass: lse and logp (packed order) for every valid row.
grpo_status run_scoring(const Layout& L, void* ws, grpo_dtype dt, const void* hidden,
                        const void* weight, int64_t N, int64_t H, int64_t V, hipStream_t s) {
  WsHeader* hdr = at<WsHeader>(ws, L.hdr);
  int32_t* rows_p = at<int32_t>(ws, L.rows);
  int32_t* y_p = at<int32_t>(ws, L.y);
  float* lse_p = at<float>(ws, L.lse);
  float* logp_p = at<float>(ws, L.logp);
  float* zy = at<float>(ws, L.zy);
  if (dt == GRPO_F32) {
    return timed(K_F32_SCORE, s, [&] {
      launch_f32_score((const float*)hidden, (const float*)weight, H, V, rows_p, y_p, hdr, lse_p,
                       logp_p, zy, N, s);
    });
  }
  float2* ms = at<float2>(ws, L.ms);
  // One launch per kScoreRows vocabulary rows: the tiles of a launch start in
  // step, while over one launch of the whole vocabulary the tiles that share
  // operand slices drift apart in K and miss in L2 (7% slower at N = 131072).
  const uint16_t* WK = weight_k(L, ws);
  for (int64_t v0 = 0; v0 < V; v0 += kScoreRows) {
    const int64_t Mc = V - v0 < kScoreRows ? V - v0 : kScoreRows;
    GemmArgs g = gemm_args(WK + (v0 / kTile) * L.sK * kTileElems, L.sK, Mc, at<uint16_t>(ws, L.hK),
                           L.sK, L.R, nullptr, &hdr->num_valid, L.Hk, nullptr);
    TRY(timed(K_GEMM_LSE, s, [&] { launch_gemm_lse(g, y_p, zy, ms, L.R, V, v0, s); }));
  }
  return timed(K_LSE_FIN, s, [&] {
    launch_lse_finalize(ms, L.R, (int)L.tiles_v, zy, hdr, lse_p, logp_p, L.R, s);
  });
}

// S7: dz recomputed per vocabulary chunk from the scoring's lse and the
// per-token g = dL/dlogp, then dL/dh = dz.W and dL/dW = dz^T.h. Shared by
// the GRPO loss and the SFT cross-entropy.
grpo_status run_backward(const Layout& L, void* ws, grpo_dtype dt, const void* hidden,
                         const void* weight, const uint8_t* mask, int64_t N, int64_t H, int64_t V,
                         void* grad_hidden, grpo_dtype grad_hidden_dt, float* grad_weight,
                         int32_t accumulate_grad_weight, hipStream_t s) {
  if (!grad_hidden && !grad_weight) return GRPO_OK;
  WsHeader* hdr = at<WsHeader>(ws, L.hdr);
  int32_t* rows_p = at<int32_t>(ws, L.rows);
  int32_t* y_p = at<int32_t>(ws, L.y);
  int32_t* pidx = at<int32_t>(ws, L.pidx);
  float* lse_p = at<float>(ws, L.lse);
  float* g_p = at<float>(ws, L.g);
  if (dt == GRPO_F32) {
    if (grad_hidden) {
      TRY(timed(K_ZERO_ROWS, s, [&] { launch_zero_masked_rows(pidx, N, H, grad_hidden, 0, s); }));
      TRY(timed(K_F32_DH, s, [&] {
        launch_f32_grad_hidden((const float*)hidden, (const float*)weight, H, V, rows_p, y_p,
                               lse_p, g_p, hdr, (float*)grad_hidden, N, s);
      }));
    }
    if (grad_weight) {
      TRY(timed(K_F32_DW, s, [&] {
        launch_f32_grad_weight((const float*)hidden, (const float*)weight, H, V, rows_p, y_p,
                               lse_p, g_p, hdr, grad_weight, accumulate_grad_weight != 0, s);
      }));
    }
    return GRPO_OK;
  }

  uint16_t* dz = at<uint16_t>(ws, L.dz);
  const uint16_t* WK = weight_k(L, ws);
  uint16_t* hK = at<uint16_t>(ws, L.hK);
  float* dhacc = L.nchunks > L.dh_group ? at<float>(ws, L.dhacc) : nullptr;
  // The tiled operands: W [V x H] and the valid hidden rows [R x H] (the
  // scoring's), and dz [R tokens x group of chunks]. dz and the chunk's W rows
  // feed the recompute natively; dL/dh reads W transposed (K = vocabulary),
  // dL/dW reads both dz and h transposed (K = tokens).
  const int64_t kt_chunk = L.sChunk, kt_h = L.sK;
  for (int64_t c = 0; c < L.nchunks; ++c) {
    int64_t v0 = c * L.Vc;
    int64_t Mc = V - v0 < L.Vc ? V - v0 : L.Vc;
    if (Mc <= 0) break;
    bool last = (c == L.nchunks - 1) || (v0 + L.Vc >= V);
    const int64_t j = c % L.dh_group;  // position of the chunk in its dL/dh group
    const int64_t vg = v0 - j * L.Vc;  // first vocabulary row of the group
    // recompute the logits of this chunk and form dz at the chunk's place in
    // the group buffer
    GemmArgs gz = gemm_args(WK + (v0 / kTile) * kt_h * kTileElems, kt_h, Mc, hK, kt_h, L.R,
                            nullptr, &hdr->num_valid, L.Hk, nullptr);
    uint16_t* dz_c = dz + j * (L.Vc / kBK) * kTileElems;
    TRY(timed(K_GEMM_DZ, s, [&] { launch_gemm_dz(gz, lse_p, g_p, dz_c, kt_chunk, V, v0, s); }));
    if (grad_weight) {
      // dW[v, :] = sum_t dz[t, v] h[t, :] over the valid tokens: A = dz and
      // B = h, both read transposed from their token-major tiled buffers
      GemmArgs gw = gemm_args(dz, kt_chunk, Mc, hK, kt_h, H, nullptr, nullptr, 0,
                              &hdr->num_valid);
      gw.a_cb0 = j * (L.Vc / kBK);
      StoreArgs sa{};
      sa.out_bf16 = 0;
      sa.out_rows = nullptr;
      sa.m_limit = Mc;
      sa.n_limit = H;
      const int splits = L.dwpart ? fill_splits((int64_t)gw.tiles_m * gw.tiles_n) : 1;
      if (splits > 1) {
        // split K: fp32 partials per split (every row/column of every tile),
        // then their sum into dW in split order
        const int64_t Hpad = round_up(H, kTile);
        gw.splits = splits;
        sa.acc_buf = at<float>(ws, L.dwpart);
        sa.ld_acc = Hpad;
        sa.split_stride = L.Vc * Hpad;
        sa.read_acc = 0;
        sa.out = nullptr;
        TRY(timed(K_GEMM_DW, s, [&] { launch_gemm_store(gw, sa, true, s); }));
        TRY(timed(K_SUM_SPLITS, s, [&] {
          launch_sum_splits(at<float>(ws, L.dwpart), splits, L.Vc * Hpad, Hpad,
                            grad_weight + v0 * H, H, Mc, H, accumulate_grad_weight != 0, s);
        }));
      } else {
        sa.acc_buf = nullptr;
        sa.ld_acc = 0;
        sa.read_acc = 0;
        sa.out = grad_weight + v0 * H;
        sa.ld_out = H;
        sa.add_out = accumulate_grad_weight != 0;
        TRY(timed(K_GEMM_DW, s, [&] { launch_gemm_store(gw, sa, true, s); }));
      }
    }
    if (grad_hidden && (j == L.dh_group - 1 || last)) {
      // dh[t, :] (+)= sum_{v in group} dz[t, v] W[v, :]: W read transposed
      GemmArgs gh = gemm_args(dz, kt_chunk, L.R, WK, kt_h, H, &hdr->num_valid, nullptr,
                              round_up(v0 + Mc - vg, kBK), nullptr);
      gh.b_kb0 = vg / kBK;
      if (L.dh_splits > 1) {  // the one dL/dh product, K split: partials, then their sum
        const int64_t Hpad = round_up(H, kTile);
        float* part = at<float>(ws, L.dhpart);
        gh.splits = L.dh_splits;
        StoreArgs sp{};
        sp.acc_buf = part;
        sp.ld_acc = Hpad;
        sp.split_stride = L.R * Hpad;
        sp.out = nullptr;
        sp.m_limit = L.R;
        sp.n_limit = H;
        TRY(timed(K_GEMM_DH, s, [&] { launch_gemm_store(gh, sp, false, s); }));
        TRY(timed(K_DH_FINISH, s, [&] {
          launch_dh_finish(part, L.dh_splits, L.R * Hpad, Hpad, hdr, L.R, H, g_p, y_p,
                           (const uint16_t*)weight, rows_p, grad_hidden,
                           grad_hidden_dt == GRPO_BF16, s);
        }));
        break;  // one product: this was the last chunk
      }
      StoreArgs sa{};
      sa.acc_buf = dhacc;
      sa.ld_acc = round_up(H, kTile);
      sa.read_acc = vg > 0;
      sa.out = last ? grad_hidden : nullptr;
      sa.ld_out = H;
      sa.out_bf16 = grad_hidden_dt == GRPO_BF16;
      if (last) {  // the sampled id's term g_t W[y_t], in fp32 before the final rounding
        sa.oh_g = g_p;
        sa.oh_y = y_p;
        sa.oh_w = (const uint16_t*)weight;
        sa.oh_ld = H;
      }
      sa.add_out = 0;
      sa.out_rows = rows_p;
      sa.m_limit = L.R;
      sa.n_limit = H;
      TRY(timed(K_GEMM_DH, s, [&] { launch_gemm_store(gh, sa, false, s); }));
    }
    if (last) break;
  }
  if (grad_weight) {  // the sampled id's term sum_{t: y_t = v} g_t h_t of dW[v], in fp32
    OnehotArgs oa;
    oa.y_p = y_p;
    oa.rows_p = rows_p;
    oa.g_p = g_p;
    oa.hdr = hdr;
    oa.hidden = (const uint16_t*)hidden;
    oa.H = H;
    oa.V = V;
    oa.n = L.R;
    for (int b = 0; b < 2; ++b) {
      oa.keys[b] = at<int32_t>(ws, L.okeys[b]);
      oa.vals[b] = at<int32_t>(ws, L.ovals[b]);
    }
    oa.counts = at<int32_t>(ws, L.ocounts);
    oa.dW = grad_weight;
    TRY(timed(K_ONEHOT, s, [&] { launch_onehot_dw(oa, s); }));
  }
  if (grad_hidden) {  // rows that packing dropped (masked, bad id or bad cu_seqlens) get dh = 0
    TRY(timed(K_ZERO_ROWS, s, [&] {
      launch_zero_masked_rows(pidx, N, H, grad_hidden, grad_hidden_dt == GRPO_BF16, s);
    }));
  }
  return GRPO_OK;
}

}  // namespace

// ======================================================================
extern "C" {

const char* grpo_status_string(grpo_status st) {
  switch (st) {
    case GRPO_OK: return "ok";
    case GRPO_ERR_NULL: return "a required pointer is NULL";
    case GRPO_ERR_SHAPE: return "a size is out of range or inconsistent";
    case GRPO_ERR_DTYPE: return "unknown or unsupported dtype";
    case GRPO_ERR_PARAM: return "a hyper-parameter is out of range";
    case GRPO_ERR_ALIGN: return "a pointer lacks the required alignment";
    case GRPO_ERR_WORKSPACE: return "workspace is NULL, misaligned or too small";
    case GRPO_ERR_DEVICE: return "no usable gfx950 device";
    case GRPO_ERR_HIP: return "a HIP runtime call failed";
    case GRPO_ERR_TOKEN_RANGE: return "a token id was outside [0, V)";
    case GRPO_ERR_SEQLENS: return "cu_seqlens was not monotone from 0 to N";
    case GRPO_ERR_CAPACITY: return "more valid rows than the workspace was sized for (max_valid)";
  }
  return "unknown status";
}

size_t grpo_workspace_bytes(grpo_op op_flags, grpo_dtype dt, int64_t N, int64_t H, int64_t V,
                            int64_t num_seqs, int64_t max_valid, size_t dz_budget) {
  const bool tiled_weight = ((int)op_flags & GRPO_WS_TILED_WEIGHT) != 0;
  const grpo_op op = (grpo_op)((int)op_flags & ~GRPO_WS_TILED_WEIGHT);
  if (op != GRPO_OP_LOGPROB_FWD && op != GRPO_OP_LOSS_FWD_BWD && op != GRPO_OP_SFT_FWD_BWD)
    return 0;
  if (tiled_weight && dt != GRPO_BF16) return 0;
  if (check_sizes(dt, N, H, V) != GRPO_OK || num_seqs < 1) return 0;
  if (max_valid < 0 || max_valid > N) return 0;
  if (op != GRPO_OP_LOGPROB_FWD && check_bwd_sizes(dt, N, H, V) != GRPO_OK) return 0;
  if (op == GRPO_OP_SFT_FWD_BWD)
    return layout(GRPO_OP_LOSS_FWD_BWD, dt, N, H, V, 1, max_valid, dz_budget, tiled_weight).total;
  return layout(op, dt, N, H, V, num_seqs, max_valid, dz_budget, tiled_weight).total;
}

size_t grpo_weight_tiled_bytes(int64_t V, int64_t H) {
  if (check_sizes(GRPO_BF16, 1, H, V) != GRPO_OK) return 0;
  return (size_t)2 * round_up(V, kTile) * tile_stride(H) * kBK;
}

grpo_status grpo_tile_weight(const void* weight, int64_t V, int64_t H, void* out,
                             size_t out_bytes, hipStream_t stream) {
  TRY(check_sizes(GRPO_BF16, 1, H, V));
  if (!weight || !out) return GRPO_ERR_NULL;
  if (!aligned(weight, 16) || !aligned(out, kAlign)) return GRPO_ERR_ALIGN;
  if (out_bytes < grpo_weight_tiled_bytes(V, H)) return GRPO_ERR_SHAPE;
  TRY(check_device());
  return timed(K_TILE, stream, [&] {
    launch_tile_rows((const uint16_t*)weight, H, nullptr, V, nullptr, round_up(V, kTile), H,
                     tile_stride(H), (uint16_t*)out, stream);
  });
}

grpo_status group_advantages(const float* rewards, int64_t num_prompts, int32_t group_size,
                             float std_eps, int32_t unbiased_std, float* adv,
                             hipStream_t stream) {
  if (!rewards || !adv) return GRPO_ERR_NULL;
  // one wave per prompt, four per 256-thread workgroup: the grid's thread
  // count stays below 2^32
  if (num_prompts < 1 || group_size < 2 || num_prompts > (1ll << 40) / group_size ||
      num_prompts > kMaxAdvPrompts)
    return GRPO_ERR_SHAPE;
  if (!(std_eps >= 0.f) || isinf(std_eps)) return GRPO_ERR_PARAM;
  TRY(check_device());
  return timed(K_ADV, stream, [&] {
    launch_group_advantages(rewards, num_prompts, group_size, std_eps, unbiased_std, adv, stream);
  });
}

grpo_status grpo_pack_valid(const uint8_t* mask, const int64_t* cu_seqlens, int64_t num_seqs,
                            int64_t N, int32_t* rows, int32_t* counts, int32_t* num_valid,
                            void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!cu_seqlens || !rows || !counts || !num_valid) return GRPO_ERR_NULL;
  if (N < 1 || N >= (1ll << 31) - kTile || num_seqs < 1 || num_seqs > N) return GRPO_ERR_SHAPE;
  Layout L = layout(GRPO_OP_LOGPROB_FWD, GRPO_F32, N, 1, 1, num_seqs, 0, 0);
  TRY(check_ws(workspace, workspace_bytes, L));
  TRY(check_device());
  return run_pack(L, workspace, mask, nullptr, 1, cu_seqlens, num_seqs, N, rows, counts,
                  num_valid, stream);
}

grpo_status grpo_pack_valid_static(const uint8_t* mask, const int64_t* cu_seqlens,
                                   int64_t num_seqs, int64_t N, int32_t* rows, int32_t* counts,
                                   int32_t* num_valid, int32_t* error_out, hipStream_t stream) {
  if (!cu_seqlens || !rows || !counts || !num_valid) return GRPO_ERR_NULL;
  if (N < 1 || N >= (1ll << 31) - kTile || num_seqs < 1 || num_seqs > N) return GRPO_ERR_SHAPE;
  if (num_seqs > kStaticMaxSeqs) return GRPO_ERR_WORKSPACE;  // beyond the static scratch
  TRY(check_device());
  char* sc = nullptr;
  TRY(static_scratch(&sc));
  PackArgs a;
  a.mask = mask;
  a.tokens = nullptr;
  a.V = 1;
  a.cu = cu_seqlens;
  a.seg = kPackSeg;
  a.B = num_seqs;
  a.N = N;
  a.counts = counts;
  a.base = (int32_t*)(sc + 256);
  a.rows_p = rows;
  a.seq_p = nullptr;
  a.y_p = nullptr;
  a.pidx = nullptr;
  a.num_valid_out = num_valid;
  a.cap = N;
  a.hdr = (WsHeader*)sc;
  TRY(timed(K_PACK, stream, [&] { launch_pack(a, stream); }));
  if (error_out)
    return timed(K_PACK, stream, [&] { launch_copy_status(a.hdr, error_out, stream); });
  return GRPO_OK;
}

grpo_status grpo_logprob_fwd(grpo_dtype dt, const void* hidden, const void* weight,
                             const void* weight_tiled, const int64_t* tokens,
                             const uint8_t* mask, int64_t N, int64_t H, int64_t V, float* logp,
                             float* lse, void* workspace, size_t workspace_bytes,
                             int64_t max_valid, hipStream_t stream) {
  TRY(check_sizes(dt, N, H, V));
  if (max_valid < 0 || max_valid > N) return GRPO_ERR_SHAPE;
  if (!hidden || !weight || !tokens) return GRPO_ERR_NULL;
  size_t al = dt == GRPO_BF16 ? 16 : 4;
  if (!aligned(hidden, al) || !aligned(weight, al) || !aligned(tokens, 8)) return GRPO_ERR_ALIGN;
  if ((logp && !aligned(logp, 4)) || (lse && !aligned(lse, 4))) return GRPO_ERR_ALIGN;
  TRY(check_weight_tiled(dt, weight_tiled));
  Layout L = layout(GRPO_OP_LOGPROB_FWD, dt, N, H, V, 1, max_valid, 0, weight_tiled != nullptr);
  L.WKx = (const uint16_t*)weight_tiled;
  TRY(check_ws(workspace, workspace_bytes, L));
  TRY(check_device());
  // one "rollout" covering every row (cu_seqlens = NULL means {0, N})
  TRY(run_pack(L, workspace, mask, tokens, V, nullptr, 1, N, nullptr, nullptr, nullptr, stream));
  if (dt == GRPO_BF16) TRY(run_tiles(L, workspace, hidden, weight, H, V, stream));
  TRY(run_scoring(L, workspace, dt, hidden, weight, N, H, V, stream));
  if (logp || lse) {
    return timed(K_LSE_FIN, stream, [&] {
      launch_rows_out(at<int32_t>(workspace, L.pidx), N, at<float>(workspace, L.logp),
                      at<float>(workspace, L.lse), logp, lse, stream);
    });
  }
  return GRPO_OK;
}

grpo_status grpo_loss_fwd_bwd(grpo_dtype dt, const void* hidden, const void* weight,
                              const void* weight_tiled, const int64_t* tokens,
                              const uint8_t* mask, const int64_t* cu_seqlens,
                              int64_t num_seqs, int64_t N, int64_t H, int64_t V,
                              const float* old_logp, const float* ref_logp,
                              const float* adv, float clip_eps, float beta, grpo_agg agg,
                              const float* lse_in, float* loss, float* logp_out, float* lse_out,
                              float* token_loss, float* dlogp, uint8_t* clip_flag,
                              void* grad_hidden, grpo_dtype grad_hidden_dt, float* grad_weight,
                              int32_t accumulate_grad_weight, void* workspace,
                              size_t workspace_bytes, int64_t max_valid, size_t dz_budget,
                              hipStream_t stream) {
  TRY(check_bwd_sizes(dt, N, H, V));
  if (max_valid < 0 || max_valid > N) return GRPO_ERR_SHAPE;
  if (!hidden || !weight || !tokens || !cu_seqlens || !old_logp || !adv || !loss)
    return GRPO_ERR_NULL;
  if (num_seqs < 1 || num_seqs > N) return GRPO_ERR_SHAPE;
  if (!(clip_eps > 0.f && clip_eps < 1.f)) return GRPO_ERR_PARAM;
  if (!(beta >= 0.f) || isinf(beta)) return GRPO_ERR_PARAM;
  if (beta != 0.f && !ref_logp) return GRPO_ERR_NULL;
  if (agg != GRPO_AGG_SEQ_MEAN && agg != GRPO_AGG_TOKEN_MEAN) return GRPO_ERR_PARAM;
  if (grad_hidden && grad_hidden_dt != GRPO_F32 && grad_hidden_dt != GRPO_BF16)
    return GRPO_ERR_DTYPE;
  if (grad_hidden && dt == GRPO_F32 && grad_hidden_dt != GRPO_F32) return GRPO_ERR_DTYPE;
  size_t al = dt == GRPO_BF16 ? 16 : 4;
  if (!aligned(hidden, al) || !aligned(weight, al) || !aligned(tokens, 8) ||
      !aligned(cu_seqlens, 8) || !aligned(old_logp, 4) || !aligned(adv, 4) || !aligned(loss, 4))
    return GRPO_ERR_ALIGN;
  if ((grad_hidden && !aligned(grad_hidden, 4)) || (grad_weight && !aligned(grad_weight, 4)))
    return GRPO_ERR_ALIGN;
  for (const void* p : {(const void*)ref_logp, (const void*)lse_in, (const void*)logp_out,
                        (const void*)lse_out, (const void*)token_loss, (const void*)dlogp})
    if (p && !aligned(p, 4)) return GRPO_ERR_ALIGN;
  TRY(check_weight_tiled(dt, weight_tiled));
  Layout L = layout(GRPO_OP_LOSS_FWD_BWD, dt, N, H, V, num_seqs, max_valid, dz_budget,
                    weight_tiled != nullptr);
  L.WKx = (const uint16_t*)weight_tiled;
  TRY(check_ws(workspace, workspace_bytes, L));
  TRY(check_device());

  void* ws = workspace;
  hipStream_t s = stream;
  WsHeader* hdr = at<WsHeader>(ws, L.hdr);
  int32_t* rows_p = at<int32_t>(ws, L.rows);
  int32_t* y_p = at<int32_t>(ws, L.y);
  int32_t* pidx = at<int32_t>(ws, L.pidx);
  float* lse_p = at<float>(ws, L.lse);
  float* logp_p = at<float>(ws, L.logp);
  float* zy = at<float>(ws, L.zy);
  float* g_p = at<float>(ws, L.g);

  // S9: pack the valid rows; per-rollout counts |o_b|.
  TRY(run_pack(L, ws, mask, tokens, V, cu_seqlens, num_seqs, N, nullptr, nullptr, nullptr, s));

  // S2-S4: scoring (or logp from a given lse).
  if (dt == GRPO_BF16 && (lse_in == nullptr || grad_hidden || grad_weight))
    TRY(run_tiles(L, ws, hidden, weight, H, V, s));
  if (lse_in == nullptr || dt == GRPO_F32) {
    TRY(run_scoring(L, ws, dt, hidden, weight, N, H, V, s));
  }
  if (lse_in != nullptr) {
    if (dt == GRPO_BF16) {
      TRY(timed(K_GATHER_DOT, s, [&] {
        launch_gather_dot_bf16((const uint16_t*)hidden, (const uint16_t*)weight, H, rows_p, y_p,
                               hdr, zy, N, s);
      }));
    }
    TRY(timed(K_LSE_FIN, s, [&] { launch_logp_from_lse(zy, lse_in, rows_p, hdr, lse_p, logp_p, N, s); }));
  }

  // S1 consumer, S5, S6: per-token objective, g = dL/dlogp, the loss.
  TokenArgs ta;
  ta.objective = 0;
  ta.N = N;
  ta.B = num_seqs;
  ta.pidx = pidx;
  ta.seq_p = at<int32_t>(ws, L.seq);
  ta.counts = at<int32_t>(ws, L.counts);
  ta.hdr = hdr;
  ta.adv = adv;
  ta.logp_p = logp_p;
  ta.lse_p = lse_p;
  ta.old_logp = old_logp;
  ta.ref_logp = beta != 0.f ? ref_logp : nullptr;
  ta.eps = clip_eps;
  ta.beta = beta;
  ta.agg = (int)agg;
  ta.g_p = g_p;
  ta.logp_out = logp_out;
  ta.lse_out = lse_out;
  ta.token_loss = token_loss;
  ta.dlogp = dlogp;
  ta.clip_flag = clip_flag;
  ta.loss_part = at<float>(ws, L.lpart);
  ta.loss = loss;
  TRY(timed(K_TOKEN, s, [&] { launch_token_objective(ta, s); }));

  if (!grad_hidden && !grad_weight) return GRPO_OK;

  // S7: gradients.
  return run_backward(L, ws, dt, hidden, weight, mask, N, H, V, grad_hidden, grad_hidden_dt,
                      grad_weight, accumulate_grad_weight, s);
}

grpo_status sft_ce_fwd_bwd(grpo_dtype dt, const void* hidden, const void* weight,
                           const void* weight_tiled, const int64_t* tokens, const uint8_t* mask,
                           int64_t N, int64_t H, int64_t V, float* loss, float* logp_out,
                           void* grad_hidden, grpo_dtype grad_hidden_dt, float* grad_weight,
                           int32_t accumulate_grad_weight, void* workspace,
                           size_t workspace_bytes, int64_t max_valid, size_t dz_budget,
                           hipStream_t stream) {
  TRY(check_bwd_sizes(dt, N, H, V));
  if (max_valid < 0 || max_valid > N) return GRPO_ERR_SHAPE;
  if (!hidden || !weight || !tokens || !loss) return GRPO_ERR_NULL;
  if (grad_hidden && grad_hidden_dt != GRPO_F32 && grad_hidden_dt != GRPO_BF16)
    return GRPO_ERR_DTYPE;
  if (grad_hidden && dt == GRPO_F32 && grad_hidden_dt != GRPO_F32) return GRPO_ERR_DTYPE;
  size_t al = dt == GRPO_BF16 ? 16 : 4;
  if (!aligned(hidden, al) || !aligned(weight, al) || !aligned(tokens, 8) || !aligned(loss, 4))
    return GRPO_ERR_ALIGN;
  if ((logp_out && !aligned(logp_out, 4)) || (grad_hidden && !aligned(grad_hidden, 4)) ||
      (grad_weight && !aligned(grad_weight, 4)))
    return GRPO_ERR_ALIGN;
  TRY(check_weight_tiled(dt, weight_tiled));
  Layout L = layout(GRPO_OP_LOSS_FWD_BWD, dt, N, H, V, 1, max_valid, dz_budget,
                    weight_tiled != nullptr);
  L.WKx = (const uint16_t*)weight_tiled;
  TRY(check_ws(workspace, workspace_bytes, L));
  TRY(check_device());
  void* ws = workspace;
  hipStream_t s = stream;

  // one "sequence" covering every row; the mask selects the supervised rows
  TRY(run_pack(L, ws, mask, tokens, V, nullptr, 1, N, nullptr, nullptr, nullptr, s));
  if (dt == GRPO_BF16) TRY(run_tiles(L, ws, hidden, weight, H, V, s));
  TRY(run_scoring(L, ws, dt, hidden, weight, N, H, V, s));

  TokenArgs ta{};
  ta.objective = 1;
  ta.N = N;
  ta.B = 1;
  ta.pidx = at<int32_t>(ws, L.pidx);
  ta.seq_p = at<int32_t>(ws, L.seq);
  ta.counts = at<int32_t>(ws, L.counts);
  ta.hdr = at<WsHeader>(ws, L.hdr);
  ta.logp_p = at<float>(ws, L.logp);
  ta.lse_p = at<float>(ws, L.lse);
  ta.g_p = at<float>(ws, L.g);
  ta.logp_out = logp_out;
  ta.loss_part = at<float>(ws, L.lpart);
  ta.loss = loss;
  TRY(timed(K_TOKEN, s, [&] { launch_token_objective(ta, s); }));
  return run_backward(L, ws, dt, hidden, weight, mask, N, H, V, grad_hidden, grad_hidden_dt,
                      grad_weight, accumulate_grad_weight, s);
}

grpo_status adamw_step(float* weight, float* exp_avg, float* exp_avg_sq, const float* grad,
                       uint16_t* weight_bf16, int64_t n, float lr, float beta1, float beta2,
                       float eps, float weight_decay, int64_t step, hipStream_t stream) {
  if (!weight || !exp_avg || !exp_avg_sq || !grad) return GRPO_ERR_NULL;
  if (n < 1 || step < 1) return GRPO_ERR_SHAPE;
  if (!(lr >= 0.f) || isinf(lr) || !(beta1 >= 0.f && beta1 < 1.f) ||
      !(beta2 >= 0.f && beta2 < 1.f) || !(eps > 0.f) || isinf(eps) || !(weight_decay >= 0.f) ||
      isinf(weight_decay))
    return GRPO_ERR_PARAM;
  if (!aligned(weight, 16) || !aligned(exp_avg, 16) || !aligned(exp_avg_sq, 16) ||
      !aligned(grad, 16) || (weight_bf16 && !aligned(weight_bf16, 8)))
    return GRPO_ERR_ALIGN;
  TRY(check_device());
  AdamArgs a;
  a.w = weight;
  a.m = exp_avg;
  a.v = exp_avg_sq;
  a.g = grad;
  a.w_bf16 = weight_bf16;
  a.n = n;
  a.beta1 = beta1;
  a.beta2 = beta2;
  a.eps = eps;
  // bias corrections in double on the host, then rounded once to fp32
  const double bc1 = 1.0 - pow((double)beta1, (double)step);
  const double bc2 = 1.0 - pow((double)beta2, (double)step);
  a.decay = (float)(1.0 - (double)lr * (double)weight_decay);
  a.step_size = (float)((double)lr / bc1);
  a.inv_sqrt_bc2 = (float)(1.0 / sqrt(bc2));
  return timed(K_ADAMW, stream, [&] { launch_adamw(a, stream); });
}

grpo_status triton_rule_reward(const uint8_t* text, int64_t text_bytes, const int64_t* offsets,
                               int64_t num_completions, const uint8_t* test_passed,
                               int32_t require_launch, int32_t weighted, float rule_weight,
                               float exec_weight, uint8_t* is_triton, float* reward,
                               hipStream_t stream) {
  if (num_completions < 0 || num_completions > 0x7fffffff || text_bytes < 0)
    return GRPO_ERR_SHAPE;
  if ((require_launch != 0 && require_launch != 1) || (weighted != 0 && weighted != 1) ||
      !isfinite(rule_weight) || !isfinite(exec_weight))
    return GRPO_ERR_PARAM;
  if (num_completions == 0) return GRPO_OK;
  if (!text || !offsets || !test_passed || !is_triton || !reward) return GRPO_ERR_NULL;
  if (!aligned(text, 16) || !aligned(offsets, 8)) return GRPO_ERR_ALIGN;
  TRY(check_device());
  RewardArgs a;
  a.text = text;
  a.text_bytes = text_bytes;
  a.offsets = offsets;
  a.test_passed = test_passed;
  a.require_launch = require_launch;
  a.weighted = weighted;
  a.w_rule = rule_weight;
  a.w_exec = exec_weight;
  a.is_triton = is_triton;
  a.reward = reward;
  return timed(K_RULE_REWARD, stream, [&] { launch_rule_reward(a, num_completions, stream); });
}

grpo_status grpo_check_error(void* workspace, hipStream_t stream) {
  if (!workspace) return GRPO_ERR_NULL;
  if (hipStreamSynchronize(stream) != hipSuccess) return GRPO_ERR_HIP;
  WsHeader h;
  if (hipMemcpy(&h, workspace, sizeof(h), hipMemcpyDeviceToHost) != hipSuccess) return GRPO_ERR_HIP;
  grpo_status st = GRPO_OK;
  if (h.err_seqlens) st = GRPO_ERR_SEQLENS;
  else if (h.err_token) st = GRPO_ERR_TOKEN_RANGE;
  else if (h.err_capacity) st = GRPO_ERR_CAPACITY;
  if (st != GRPO_OK) {
    h.err_seqlens = h.err_token = h.err_capacity = 0;
    if (hipMemcpy(workspace, &h, 4 * sizeof(int32_t), hipMemcpyHostToDevice) != hipSuccess)
      return GRPO_ERR_HIP;
  }
  return st;
}

void grpo_profile_enable(int32_t on) {
  Prof& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  p.on = on != 0;
}

void grpo_profile_reset(void) {
  Prof& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  for (auto& r : p.recs) {
    (void)hipEventSynchronize(r.b);
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  p.recs.clear();
  for (int k = 0; k < K_NUM_KINDS; ++k) {
    p.launches[k] = 0;
    p.ms[k] = 0.0;
  }
}

int32_t grpo_profile_num_kinds(void) { return K_NUM_KINDS; }

const char* grpo_profile_kind_name(int32_t kind) {
  if (kind < 0 || kind >= K_NUM_KINDS) return "";
  return kKindNames[kind];
}

grpo_status grpo_profile_query(int32_t kind, int64_t* launches, double* total_ms) {
  if (kind < 0 || kind >= K_NUM_KINDS) return GRPO_ERR_PARAM;
  if (!launches || !total_ms) return GRPO_ERR_NULL;
  Prof& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  TRY(fold_records(p));
  *launches = p.launches[kind];
  *total_ms = p.ms[kind];
  return GRPO_OK;
}

}  // extern "C"
