// bf16 MFMA contraction C[m, n] = sum_k A[m, k] * B[n, k] for gfx950, with
// fused epilogues for the four products of the GRPO path:
//
//   EpiLse        forward scoring: A = LM-head rows (vocabulary), B = hidden
//                 rows (tokens). Reduces each token column of the 256x256 tile
//                 to online (max, sum-exp) partials and picks out z at the
//                 sampled id.
//   EpiDz         backward: the same tile recomputed and turned into
//                 dz = -g * exp(z - lse), stored in bf16 token-major (the
//                 sampled id's +g is applied in fp32 by the two products below
//                 and by the one-hot kernel).
//   EpiGradHidden dL/dh = dz . W, and EpiGradWeight dL/dW = dz^T . h: fp32
//                 stores, optionally accumulating, gathering output rows,
//                 converting to bf16, or adding the sampled id's term.
//
// Tiling: one 256-thread workgroup (four waves, one per SIMD) per 256x256
// output tile, K in steps of 32 from operands in the library's tiled layout
// (see the main loop).
//
// Tile order: workgroup ids are dealt round-robin to the 8 XCDs, so id
// b runs on XCD b % 8. Tiles are assigned so that each XCD owns a band of
// kGM tile-rows and walks the tile-columns in blocks of kGN, and all 8 XCDs
// walk the same columns at the same time: the B operand is then shared
// through the last-level cache and each XCD's L2 sees only kGM + kGN
// distinct operand slices per K step. Tile-rows after the last whole group
// of 8 bands are shared out evenly over the XCDs; products with fewer than
// 8 kGM tile-rows split the valid tile-columns among the XCDs instead. A
// product may also split K over the grid's y dimension (partial sums to a
// buffer).
#include "kernels.h"

namespace grpo {

#ifndef GRPO_GEMM_GM
#define GRPO_GEMM_GM 4
#endif
#ifndef GRPO_GEMM_GN
#define GRPO_GEMM_GN 8
#endif
constexpr int kGM = GRPO_GEMM_GM;  // tile-rows per XCD band
constexpr int kGN = GRPO_GEMM_GN;  // tile-columns per step of the walk
// s_waitcnt immediate: vmcnt <= n (6 bits, split over [3:0] and [15:14]),
// expcnt left at its maximum (7 in [6:4]), lgkmcnt 0 ([11:8]).
constexpr int wait_vm(int n) { return (n & 15) | ((n >> 4) << 14) | 0x0070; }

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4* lds_i16x4_ptr_t;

// Operand loads go global -> LDS through a buffer resource based at the
// tile-row's first block: each lane's offset is fixed, the K step goes in the
// scalar offset, and one instruction moves 16 bytes per lane (1 KiB of
// consecutive LDS at M0). Offsets stay far below 4 GiB (a tile-row of the
// largest operand, 2^20 columns, is 512 MiB); the range check is off.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const uint16_t* base) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, -1, 0x00020000);
}
__device__ __forceinline__ void load_lds16(__amdgpu_buffer_rsrc_t r, char* lds, uint32_t voff,
                                           uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)lds, 16, voff, soff, 0, 0);
}
// The same load issued from inline assembly, for kernels that read LDS with
// ds_read_b64_tr_b16: the compiler cannot tell those reads apart from the
// loads' LDS destinations and would wait for every load in flight before each
// of them. Here the compiler sees no load at all, so the kernel itself waits
// (vmcnt) before LDS that a load writes is read or reused. M0 is set in the
// same statement; no other code of these kernels uses it. The resource and
// the scalar offset must be values the compiler holds in scalar registers
// (wave-uniform); where it does not, the assembler rejects the instruction,
// so such a change fails the build rather than the run.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void load_lds16_asm(__amdgpu_buffer_rsrc_t r, uint32_t lds,
                                               uint32_t voff, uint32_t soff) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane(lds);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :
               : "s"(m0), "v"(voff), "s"(r), "s"(soff)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// Maps a workgroup id to its (tile_m, tile_n); returns false for the
// padding workgroups of the last band. With fewer than 8 kGM tile-rows there
// are not enough rows for a band per XCD (column_tile_of).
__device__ inline bool tile_of(int bid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int xcd = bid & 7, loc = bid >> 3;
  const int per_band = kGM * tiles_n;
  const int full = tiles_m / (8 * kGM);  // whole groups of 8 bands
  const int band = loc / per_band;
  if (band < full) {
    const int r = loc - band * per_band;
    const int nb = r / (kGM * kGN);
    const int r2 = r - nb * (kGM * kGN);
    tm = band * (8 * kGM) + xcd * kGM + r2 % kGM;
    tn = nb * kGN + r2 / kGM;
    return true;
  }
  // The rem tile-rows after them are shared out so that the XCDs get equal
  // work: from 8 rows on, each XCD takes rem/8 or rem/8 + 1 consecutive rows
  // and walks them kGN columns at a time; below 8, each XCD takes an eighth
  // of the columns over all rem rows.
  const int rem = tiles_m - full * (8 * kGM);
  const int l = loc - full * per_band;
  if (rem == 0) return false;
  if (rem >= 8) {
    const int q = rem >> 3, e = rem & 7;
    const int cnt = q + (xcd < e ? 1 : 0);
    const int nb = l / (cnt * kGN), r2 = l - nb * (cnt * kGN);
    tm = full * (8 * kGM) + xcd * q + min(xcd, e) + r2 % cnt;
    tn = nb * kGN + r2 / cnt;
    return tn < tiles_n;
  }
  const int cols = (tiles_n + 7) >> 3;
  if (l >= rem * cols) return false;
  tm = full * (8 * kGM) + l % rem;
  tn = xcd * cols + l / rem;
  return tn < tiles_n;
}

// Few tile-rows: each XCD takes an eighth of the tile-columns that hold valid
// columns (tiles_n, known only on the device when the column count is), all
// rows, walking them column by column; false for workgroups without a tile.
__device__ inline bool column_tile_of(int bid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int xcd = bid & 7, loc = bid >> 3;
  const int cols = (tiles_n + 7) >> 3;  // tile-columns per XCD
  if (loc >= tiles_m * cols) return false;
  tm = loc % tiles_m;
  tn = xcd * cols + loc / tiles_m;
  return tn < tiles_n;
}

// Tile-rows that make 1, 2 or 4 whole bands: the 8 XCDs are shared out over
// the bands (8, 4 or 2 per band), each band's tile-columns over its XCDs, and
// each XCD walks its part of its band as tile_of does.
__host__ __device__ inline bool split_bands(int tiles_m) {
  return tiles_m < 8 * kGM && tiles_m % kGM == 0 && 8 % (tiles_m / kGM) == 0;
}
__host__ __device__ inline int split_band_cols(int tiles_m, int tiles_n) {
  const int parts = 8 / (tiles_m / kGM);
  return (tiles_n + parts - 1) / parts;  // tile-columns per XCD
}
__device__ inline bool split_band_tile_of(int bid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int xcd = bid & 7, loc = bid >> 3;
  const int bands = tiles_m / kGM;
  const int cols = split_band_cols(tiles_m, tiles_n);
  const int nb = loc / (kGM * kGN), r2 = loc - nb * (kGM * kGN);
  const int c = nb * kGN + r2 / kGM;
  tm = (xcd % bands) * kGM + r2 % kGM;
  tn = (xcd / bands) * cols + c;
  return c < cols && tn < tiles_n;
}

// Tile of this workgroup, or false if it has none (or only rows or columns
// past the valid counts). The mapping is chosen by the grid's tile-rows.
__device__ inline bool gemm_tile(const GemmArgs& g, int m_valid, int n_valid, int& tm, int& tn) {
  if (split_bands(g.tiles_m))
    return split_band_tile_of(blockIdx.x, g.tiles_m, g.tiles_n, tm, tn) && tm * kTile < m_valid &&
           tn * kTile < n_valid;
  if (g.tiles_m < 8 * kGM) {
    if (m_valid <= 0 || n_valid <= 0) return false;
    return column_tile_of(blockIdx.x, min(g.tiles_m, (int)ceil_div(m_valid, kTile)),
                          min(g.tiles_n, (int)ceil_div(n_valid, kTile)), tm, tn);
  }
  return tile_of(blockIdx.x, g.tiles_m, g.tiles_n, tm, tn) && tm * kTile < m_valid &&
         tn * kTile < n_valid;
}

int gemm_grid(int tiles_m, int tiles_n) {
  if (split_bands(tiles_m)) return 8 * kGM * (int)round_up(split_band_cols(tiles_m, tiles_n), kGN);
  if (tiles_m < 8 * kGM) return 8 * tiles_m * (int)ceil_div(tiles_n, 8);
  // workgroups per XCD: the whole groups of bands, then the rows tile_of
  // shares out after them
  const int full = tiles_m / (8 * kGM), rem = tiles_m % (8 * kGM);
  int tail = 0;
  if (rem >= 8)
    tail = ((rem + 7) / 8) * kGN * (int)ceil_div(tiles_n, kGN);
  else if (rem > 0)
    tail = rem * (int)ceil_div(tiles_n, 8);
  return 8 * (full * kGM * tiles_n + tail);
}

// ------------------------------------------------------------ layout
// Wave w (one per SIMD) owns rows (w%2)*128 and columns (w/2)*128 of the tile
// as 8 x 8 blocks of v_mfma_f32_16x16x32_bf16 (64 x 4 fp32 accumulators per
// lane, in AGPRs). Register r of block (i, j) of lane l holds row
// i*16 + (l/16)*4 + r and column j*16 + l%16 of the wave's part. Per flop this
// MFMA shape moves half the accumulator data of v_mfma_f32_32x32x16_bf16,
// which lets the part hold a higher clock under its power limit (1.8 vs 1.5
// GHz on these products, the MFMA units equally busy).
struct Frag {
  int tm, tn, wm, wn, lane;
  // row (within the tile) of register r of block row i, and column of block column j
  __device__ int row(int i, int r) const { return wm * 128 + i * 16 + (lane >> 4) * 4 + r; }
  __device__ int col(int j) const { return wn * 128 + j * 16 + (lane & 15); }
};
typedef f32x4 Acc[8][8];

// Forward scoring: A = vocabulary rows, B = tokens. Each token column of a
// wave's 128-row half tile is spread over four lanes (32 rows each); each lane
// reduces its rows to (max, sum exp(z - max)), the four partials are merged by
// two cross-lane exchanges, the two half tiles through LDS, and the tile
// writes one partial per token. z at the sampled id is taken from the
// accumulator.
struct EpiLse {
  static constexpr bool kKPositive = true;  // K = H >= 32
  const int32_t* y_p;  // sampled id of each packed token
  float* zy;           // z at the sampled id, per packed token
  float2* ms;          // [tiles of V][ldms] partial (max, sum-exp) per tile and token
  int64_t ldms;
  int64_t V;
  int64_t v0;          // first vocabulary row of this launch (a multiple of 256)

  // the sampled id of each column of this lane, loaded before the main loop so
  // that the loop hides its latency (the per-token arrays hold a value for
  // every column of the grid; those past the valid tokens are ignored)
  struct Pre {
    int y[8];
  };
  __device__ __forceinline__ Pre prefetch(const Frag& f) const {
    Pre p;
    static_for<8>([&](auto j) { p.y[j] = y_p[(int64_t)f.tn * kTile + f.col(j)]; });
    return p;
  }

  // (max, sum exp(z - max)) of this lane's 32 rows of column j (row offsets
  // i*16 + r; those >= vlim are past the vocabulary); z at row offset y
  template <bool FULL, class J>
  __device__ __forceinline__ void column(const Acc& acc, J j, float& m_out, float& s_out,
                                         int vlim, int y, float* zy_t) const {
    float m = -INFINITY;
    static_for<8>([&](auto i) {
      static_for<4>([&](auto r) {
        if (FULL || i * 16 + r < vlim) m = fmaxf(m, acc[i][j][r.value]);
      });
    });
    float sum = 0.f;
    const float m2l = m * kLog2e;
    static_for<8>([&](auto i) {
      static_for<4>([&](auto r) {
        if (FULL || i * 16 + r < vlim)
          sum += __builtin_amdgcn_exp2f(fmaf(acc[i][j][r.value], kLog2e, -m2l));
      });
    });
    // the lane holding the sampled id's row (offsets i*16 + r, r < 4)
    if ((unsigned)y < 128u && (y & 12) == 0) {
      float z = 0.f;
      static_for<8>([&](auto i) {
        static_for<4>([&](auto r) {
          if (i * 16 + r == y) z = acc[i][j][r.value];
        });
      });
      *zy_t = z;
    }
    m_out = m;
    s_out = sum;
  }

  // merges (m2, s2) into (m, s); an empty partial is (-inf, 0)
  static __device__ __forceinline__ void merge2(float& m, float& s, float m2, float s2) {
    const float mm = fmaxf(m, m2);
    s = (s == 0.f ? 0.f : s * __expf(m - mm)) + (s2 == 0.f ? 0.f : s2 * __expf(m2 - mm));
    m = mm;
  }
  static __device__ __forceinline__ void merge(float& m, float& s, int lanes) {
    merge2(m, s, __shfl_xor(m, lanes, 64), __shfl_xor(s, lanes, 64));
  }

  __device__ __forceinline__ void operator()(Acc& acc, const Frag& f, int, int n_valid,
                                             char* smem, const Pre& pre) const {
    const int64_t tile_v = v0 / kTile + f.tm;  // this tile's index over the vocabulary
    const int64_t vbase = tile_v * kTile + f.row(0, 0);
    const int vlim = (int)(V - vbase);  // row offset o of this lane is valid iff o < vlim
    const bool full = tile_v * kTile + f.wm * 128 + 128 <= V;  // wave-uniform
    float pm[8], ps[8];
    static_for<8>([&](auto j) {
      const int64_t t = (int64_t)f.tn * kTile + f.col(j);
      const int y = t < n_valid ? (int)(pre.y[j] - vbase) : -1;  // y as a row offset of this lane
      if (full)
        column<true>(acc, j, pm[j], ps[j], vlim, y, zy + t);
      else
        column<false>(acc, j, pm[j], ps[j], vlim, y, zy + t);
      merge(pm[j], ps[j], 16);
      merge(pm[j], ps[j], 32);
      __builtin_amdgcn_sched_barrier(0);  // one column at a time (bounds live registers)
    });
    // the two waves of a column block (rows 0-127 and 128-255) merge into one
    // partial per token: the lower half's wave adds the upper half's (fixed order)
    float2* xchg = (float2*)smem + f.wn * 128;
    if (f.wm == 1 && f.lane < 16)
      static_for<8>([&](auto j) { xchg[j * 16 + f.lane] = make_float2(pm[j], ps[j]); });
    __syncthreads();
    if (f.wm == 0 && f.lane < 16) {
      static_for<8>([&](auto j) {
        const int64_t t = (int64_t)f.tn * kTile + f.col(j);
        const float2 u = xchg[j * 16 + f.lane];
        merge2(pm[j], ps[j], u.x, u.y);
        if (t < n_valid) ms[tile_v * ldms + t] = make_float2(pm[j], ps[j]);
      });
    }
  }
};

// Backward: the tile recomputed and turned into dz = -g * exp(z - lse) (the
// sampled id's +g is applied exactly in fp32 by the callers of the two
// gradient products), stored in bf16, token-major: the dL/dh product reads it
// as is, the dL/dW product through transposing LDS reads.
struct EpiDz {
  static constexpr bool kKPositive = true;  // K = H >= 32
  const float* lse_p;
  const float* g_p;
  uint16_t* dz;    // tiled [tokens][chunk vocabulary], dz_kt 32-wide blocks per tile-row
  int64_t dz_kt;
  int64_t V;       // vocabulary size
  int64_t v0;      // first vocabulary row of this chunk

  // lse and g of each column of this lane, loaded before the main loop
  struct Pre {
    float lse[8], g[8];
  };
  __device__ __forceinline__ Pre prefetch(const Frag& f) const {
    Pre p;
    static_for<8>([&](auto j) {
      const int64_t t = (int64_t)f.tn * kTile + f.col(j);
      p.lse[j] = lse_p[t];
      p.g[j] = g_p[t];
    });
    return p;
  }

  __device__ __forceinline__ void operator()(Acc& acc, const Frag& f, int, int n_valid, char*,
                                             const Pre& pre) const {
    const int64_t vbase = v0 + (int64_t)f.tm * kTile + f.row(0, 0);
    const int vlim = (int)((V - vbase) < (1 << 20) ? (V - vbase) : (1 << 20));
    const bool full = v0 + (int64_t)f.tm * kTile + f.wm * 128 + 128 <= V;  // wave-uniform
    if (full)
      body(acc, f, pre, n_valid, vlim, std::true_type{});
    else
      body(acc, f, pre, n_valid, vlim, std::false_type{});
  }

  // -g * p of this lane's values in bf16: the four rows i*16 + (l/16)*4 .. +3 of
  // column j are 8 consecutive bytes of token row j*16 + l%16 of the tiled
  // token-major buffer (each store instruction covers 16 rows x 32 bytes)
  template <class Full>
  __device__ __forceinline__ void body(Acc& acc, const Frag& f, const Pre& pre, int n_valid,
                                       int vlim, Full) const {
    const int q = f.lane >> 4;
    // block (token tile-row tn, vocabulary block tm*8 + wm*4 + i/2), row
    // wn*128 + j*16 + l%16, column (i%2)*16 + q*4
    uint16_t* base = dz + ((int64_t)f.tn * dz_kt + f.tm * 8 + f.wm * 4) * kTileElems +
                     (f.wn * 128 + (f.lane & 15)) * kBK + q * 4;
    static_for<8>([&](auto j) {
      const int64_t t = (int64_t)f.tn * kTile + f.col(j);
      const bool tv = t < n_valid;
      // p = exp(z - lse) = exp2(z*log2e - lse*log2e); invalid columns get g = 0
      const float l2 = tv ? pre.lse[j] * kLog2e : 0.f;
      const float ng = tv ? -pre.g[j] : 0.f;
      static_for<8>([&](auto i) {
        float d[4];
        static_for<4>([&](auto r) {
          const float v = ng * __builtin_amdgcn_exp2f(fmaf(acc[i][j][r.value], kLog2e, -l2));
          d[r] = (Full::value || i * 16 + r < vlim) ? v : 0.f;
        });
        *(uint2*)(base + (i / 2) * kTileElems + j * 16 * kBK + (i % 2) * 16) =
            make_uint2(bf16_pack2(d[0], d[1]), bf16_pack2(d[2], d[3]));
      });
      __builtin_amdgcn_sched_barrier(0);  // one column at a time (bounds live registers)
    });
  }
};

// fp32 store epilogue on the 16x16 layout; optionally adds, to every row m
// of the output, oh_g[m] times row oh_y[m] of the bf16 matrix oh_w (the
// sampled id's term of dL/dh, kept out of the bf16 dz operand).
struct EpiStore {
  static constexpr bool kKPositive = false;  // dL/dW over no valid tokens, empty K splits
  StoreArgs s;

  struct Pre {};
  __device__ __forceinline__ Pre prefetch(const Frag&) const { return {}; }

  __device__ __forceinline__ void operator()(Acc& acc, const Frag& f, int m_valid, int,
                                             char*, const Pre&) const {
    const int64_t mlim = s.m_limit < m_valid ? s.m_limit : m_valid;
    const int64_t m0 = (int64_t)f.tm * kTile + f.row(0, 0);
    const int64_t n0 = (int64_t)f.tn * kTile + f.col(0);
    const bool full = (int64_t)f.tm * kTile + kTile <= mlim &&
                      (int64_t)f.tn * kTile + kTile <= s.n_limit;
    float* pacc = s.acc_buf ? s.acc_buf + blockIdx.y * s.split_stride + m0 * s.ld_acc + n0 : nullptr;
    // one block row (4 rows x 8 columns of this lane) at a time: loaded,
    // combined and stored before the next starts
    static_for<8>([&](auto i) {
      float v[4][8];
      static_for<4>([&](auto r) { static_for<8>([&](auto j) { v[r][j] = acc[i][j][r.value]; }); });
      if (s.read_acc) {
        float prev[4][8];
        static_for<4>([&](auto r) {
          const float* pr = pacc + (i * 16 + r) * s.ld_acc;
          static_for<8>([&](auto j) { prev[r][j] = pr[j * 16]; });
        });
        static_for<4>([&](auto r) { static_for<8>([&](auto j) { v[r][j] += prev[r][j]; }); });
      }
      if (s.oh_g != nullptr) {
        static_for<4>([&](auto r) {
          const int64_t m = m0 + i * 16 + r;
          if (full || m < mlim) {
            const float gm = s.oh_g[m];
            const uint16_t* wr = s.oh_w + (int64_t)s.oh_y[m] * s.oh_ld + n0;
            static_for<8>([&](auto j) {
              if (full || n0 + j * 16 < s.n_limit) v[r][j] += gm * bf16_bits_to_f32(wr[j * 16]);
            });
          }
        });
      }
      if (s.out == nullptr) {
        static_for<4>([&](auto r) {
          float* pr = pacc + (i * 16 + r) * s.ld_acc;
          static_for<8>([&](auto j) { pr[j * 16] = v[r][j]; });
        });
      } else if (full) {
        int64_t orow[4];
        static_for<4>([&](auto r) {
          const int64_t m = m0 + i * 16 + r;
          orow[r] = (s.out_rows ? (int64_t)s.out_rows[m] : m) * s.ld_out + n0;
        });
        if (s.out_bf16) {
          uint16_t* ob = (uint16_t*)s.out;
          static_for<4>([&](auto r) {
            static_for<8>([&](auto j) { ob[orow[r] + j * 16] = bf16_bits(v[r][j]); });
          });
        } else {
          float* of = (float*)s.out;
          if (s.add_out) {
            float prev[4][8];
            static_for<4>([&](auto r) {
              static_for<8>([&](auto j) { prev[r][j] = of[orow[r] + j * 16]; });
            });
            static_for<4>([&](auto r) { static_for<8>([&](auto j) { v[r][j] += prev[r][j]; }); });
          }
          static_for<4>([&](auto r) {
            static_for<8>([&](auto j) { of[orow[r] + j * 16] = v[r][j]; });
          });
        }
      } else {  // edge tile: per-element bounds
        static_for<4>([&](auto r) {
          const int64_t m = m0 + i * 16 + r;
          if (m < mlim) {
            const int64_t orow = s.out_rows ? (int64_t)s.out_rows[m] : m;
            static_for<8>([&](auto j) {
              const int64_t n = n0 + j * 16;
              if (n < s.n_limit) {
                if (s.out_bf16) {
                  ((uint16_t*)s.out)[orow * s.ld_out + n] = bf16_bits(v[r][j]);
                } else {
                  float* o2 = (float*)s.out + orow * s.ld_out + n;
                  *o2 = s.add_out ? *o2 + v[r][j] : v[r][j];
                }
              }
            });
          }
        });
      }
      __builtin_amdgcn_sched_barrier(0);
    });
  }
};
struct EpiGradHidden : EpiStore {};
struct EpiGradWeight : EpiStore {};

// ------------------------------------------------------------ main loop
// Both operands are in the tiled layout: tile-row r of an operand is a run
// of 256 x 32 blocks (16 KiB each, rows of 64 bytes), block kb of it at
// (r * kt + kb0 + kb) * 8192 elements. One K step (32) of a tile is then one
// contiguous 16 KiB block per operand, and each 1 KiB load instruction of a
// wave covers eight whole 128-byte lines.
//
// LDS is a ring of 5 stages of 32 KiB (A block + B block of one K step),
// filled by loads that go straight from global memory to LDS. A step is 64
// MFMAs per wave on 8 A and 8 B fragments held in registers; the fragments of
// step kt+1 are read during the first 16 MFMAs of step kt, and the 8 loads of
// step kt+5 are spread over its MFMAs. The barrier at the end of step kt
// (after every wave's reads of step kt+1 have returned and its loads of step
// kt+2 have landed) frees the stage of step kt+1. 16-byte chunks of a stage
// row are XOR-swizzled by row bits 1-2, which keeps both the fragment reads
// (16 rows x 4 chunks per instruction) and the loads free of bank conflicts.
// The fragment reads of one K step as a list of instructions: fragments in
// the order the step's MFMAs first use them (A0, B0..B7, A1..A7), a
// transposed operand's fragment as its two halves. q(k) is the fragment of
// instruction k, part(k) -1 for a whole fragment, else the half.
template <bool TA, bool TB>
struct ReadSchedule {
  static constexpr int frag_at(int n) { return n == 0 ? 0 : n <= 8 ? n + 7 : n - 8; }
  static constexpr int width(int q) { return (q < 8 ? TA : TB) ? 2 : 1; }
  static constexpr int kOps = 8 * width(0) + 8 * width(8);
  static constexpr int q(int k) {
    for (int n = 0; n < 16; ++n) {
      if (k < width(frag_at(n))) return frag_at(n);
      k -= width(frag_at(n));
    }
    return -1;
  }
  static constexpr int part(int k) {
    for (int n = 0; n < 16; ++n) {
      const int wd = width(frag_at(n));
      if (k < wd) return wd == 1 ? -1 : k;
      k -= wd;
    }
    return -1;
  }
};

constexpr int kWaves = 4;
constexpr int kStage = 2 * kTileElems * 2;              // bytes of one A + B stage
constexpr int kStages = 5;
constexpr int kJ = kTileElems * 2 / 1024 / kWaves;      // 1 KiB loads per operand per wave per step

template <class Epi, bool TA, bool TB>
__global__ void __launch_bounds__(256, 1) k_gemm(GemmArgs g, Epi epi) {
  __shared__ __attribute__((aligned(16))) char smem[kStages * kStage];
  const int m_valid = g.m_dev ? min(*g.m_dev, g.M) : g.M;
  const int n_valid = g.n_dev ? min(*g.n_dev, g.N) : g.N;
  int tm, tn;
  if (!gemm_tile(g, m_valid, n_valid, tm, tn)) return;
  // this workgroup's part of K: blocks [kb0, kb0 + K/32) of an even split
  // over the grid's y dimension (a part past the end does no K steps)
  int K = g.k_dev ? (int)round_up(*g.k_dev, kBK) : g.K;
  int64_t kb0 = 0;
  if (g.splits > 1) {
    const int per = (int)ceil_div(K / kBK, g.splits);
    const int first = (int)blockIdx.y * per;
    const int cnt = K / kBK - first < per ? K / kBK - first : per;
    kb0 = cnt > 0 ? first : 0;
    K = cnt > 0 ? cnt * kBK : 0;
  }

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = w & 1, wn = w >> 1;
  const Frag f{tm, tn, wm, wn, lane};
  const auto pre = epi.prefetch(f);

  Acc acc;
  static_for<8>([&](auto i) {
    static_for<8>([&](auto j) { acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f}; });
  });

  // ---- loads: the j-th load of lane l of wave w fills stage row
  // q = 16*(w + 4j) + l/4 at physical chunk l%4, i.e. logical chunk
  // (l%4) ^ ((q/2)%4); one instruction writes 1 KiB of consecutive LDS.
  const int qrow = 16 * w + (lane >> 2);
  const int qch = (lane & 3) ^ ((qrow >> 1) & 3);
  const __amdgpu_buffer_rsrc_t ra =
      tile_rsrc(g.A + ((int64_t)tm * g.a_kt + g.a_kb0 + kb0) * kTileElems);
  const __amdgpu_buffer_rsrc_t rb =
      tile_rsrc(g.B + ((int64_t)tn * g.b_kt + g.b_kb0 + kb0) * kTileElems);
  const uint32_t lofs = (uint32_t)(qrow * 32 + qch * 8) * 2;
  // A transposed operand's K step is 32 rows of its 8 column blocks: 8 runs of
  // 2 KiB, each row 64 contiguous bytes. Load j (of 16) moves rows 16 (j%2)
  // .. +15 of column block j/2 into stage bytes j * 1024; the buffer resource
  // is rebased on every step (K crosses block-rows every 8 steps). A row r
  // with bit 1 xor bit 3 set holds its two 32-byte halves swapped (lane l of
  // a load fills row l/4 of its 16, physical chunk l%4), so that the rows of a
  // transposing read spread over all banks (see the fragment reads).
  const int tsw = ((lane >> 3) ^ (lane >> 5)) & 1;
  const int tsrc = (lane & ~3) * 8 + ((lane & 3) ^ (tsw << 1)) * 8;
  const uint32_t tofs[kJ] = {
      (uint32_t)(((w >> 1) * 8192 + (w & 1) * 512 + tsrc) * 2),
      (uint32_t)((((w + 4) >> 1) * 8192 + (w & 1) * 512 + tsrc) * 2),
      (uint32_t)((((w + 8) >> 1) * 8192 + (w & 1) * 512 + tsrc) * 2),
      (uint32_t)((((w + 12) >> 1) * 8192 + (w & 1) * 512 + tsrc) * 2)};
  auto trsrc = [&](const uint16_t* X, int64_t x_kt, int64_t x_kb0, int64_t x_cb0, int t, int kt) {
    const int64_t kr = (x_kb0 + kb0 + kt) * kBK;  // first storage row of this K step
    return tile_rsrc(X + (((kr >> 8) * x_kt + x_cb0 + (int64_t)t * 8) * kTileElems +
                          (kr & 255) * kBK));
  };
  // LDS address of smem (the kernel's only LDS object, so in practice 0)
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)smem;
  auto ld = [&](__amdgpu_buffer_rsrc_t r, char* lds, uint32_t voff, uint32_t soff) {
    if constexpr (TA || TB)
      load_lds16_asm(r, lds0 + (uint32_t)(lds - smem), voff, soff);
    else
      load_lds16(r, lds, voff, soff);
  };
  auto load = [&](int kt, char* la, auto l) {
    const uint32_t so = (uint32_t)kt * (kTileElems * 2);
    if constexpr (l.value < kJ) {
      if constexpr (TA)
        ld(trsrc(g.A, g.a_kt, g.a_kb0, g.a_cb0, tm, kt), la - w * 1024 + (w + 4 * l.value) * 1024,
           tofs[l.value], 0);
      else
        ld(ra, la + l.value * 1024 * kWaves, lofs + l.value * 16 * kWaves * 64, so);
    } else {
      if constexpr (TB)
        ld(trsrc(g.B, g.b_kt, g.b_kb0, g.b_cb0, tn, kt),
           la - w * 1024 + kTileElems * 2 + (w + 4 * (l.value - kJ)) * 1024, tofs[l.value - kJ], 0);
      else
        ld(rb, la + kTileElems * 2 + (l.value - kJ) * 1024 * kWaves,
           lofs + (l.value - kJ) * 16 * kWaves * 64, so);
    }
  };
  auto load_step = [&](int kt, int stage) {
    char* la = smem + stage * kStage + w * 1024;
    static_for<2 * kJ>([&](auto l) { load(kt, la, l); });
  };

  // ---- fragments of one step: q < 8 A block q, else B block q - 8
  const int fr = lane & 15;
  const int rch = ((lane >> 4) ^ ((fr >> 1) & 3)) << 4;
  const int rd_a = (wm * 128 + fr) * 64 + rch;
  const int rd_b = kTileElems * 2 + (wn * 128 + fr) * 64 + rch;
  // A transposed operand's fragment: two transposing reads (ds_read_b64_tr_b16:
  // within 16 lanes, lane i receives element i%4 of the 8 bytes lanes i/4,
  // 4 + i/4, 8 + i/4, 12 + i/4 address). Lane a of 16-lane group g addresses
  // row 8g + 4r + a/4 and the 4 columns 4 (a%4) .. +3 of the block's 16, so
  // that lane i gets K rows 8g + 4r .. +3 of column i; r = 0, 1 give 8 rows.
  // A group's 16 lanes read 4 rows x 32 bytes, two groups 8 rows: with the
  // halves swapped on bit 1 xor bit 3 of the row, the 4 rows fall on distinct
  // 32-byte quarters of 128 bytes of banks and the 8 rows on distinct eighths
  // of 256 bytes.
  const int tr_row = 8 * (lane >> 4) + ((lane & 15) >> 2);
  const int tr_sw = (((lane >> 3) ^ (lane >> 4)) & 1) * 32;  // bit 1 ^ bit 3 of tr_row
  const int tr_a = tr_row * 64 + (lane & 3) * 8 + wm * 4 * 2048;
  const int tr_b = kTileElems * 2 + tr_row * 64 + (lane & 3) * 8 + wn * 4 * 2048;
  const int tr_h[2] = {tr_sw, 32 - tr_sw};  // byte offset of half 0 / half 1
  bf16x8 fs[2][16];
  i16x4 fh[2][16][2];  // the halves of a transposed operand's fragments
  // part: -1 the whole fragment, 0 / 1 one half of a transposed fragment
  auto fread = [&](auto slot, auto st, auto q, auto part) {
    const char* base = smem + st.value * kStage;
    constexpr bool T = q.value < 8 ? TA : TB;
    if constexpr (T) {
      constexpr int blk = q.value % 8;  // column block blk/2 of the wave's four, half blk%2
      const char* pr = base + (q.value < 8 ? tr_a : tr_b) + tr_h[blk % 2] + (blk / 2) * 2048;
      static_for<2>([&](auto r) {
        if constexpr (part.value < 0 || part.value == r.value)
          fh[slot.value][q.value][r.value] =
              __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_ptr_t)(pr + r.value * 4 * 64));
      });
    } else if constexpr (q.value < 8) {
      fs[slot.value][q.value] = *(const bf16x8*)(base + rd_a + q.value * 16 * 64);
    } else {
      fs[slot.value][q.value] = *(const bf16x8*)(base + rd_b + (q.value - 8) * 16 * 64);
    }
  };
  // MFMA m of a step: block row i = m/8, block column j in a snake order
  // (each MFMA changes one operand from the one before)
  auto frag = [&](auto slot, auto q) {
    constexpr bool T = q.value < 8 ? TA : TB;
    if constexpr (T)
      return __builtin_bit_cast(bf16x8, __builtin_shufflevector(fh[slot.value][q.value][0],
                                                                fh[slot.value][q.value][1], 0, 1,
                                                                2, 3, 4, 5, 6, 7));
    else
      return fs[slot.value][q.value];
  };
  auto mfma = [&](auto slot, auto m) {
    constexpr int i = m.value / 8, jj = m.value % 8, j = (i & 1) ? 7 - jj : jj;
    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
        frag(slot, std::integral_constant<int, i>{}),
        frag(slot, std::integral_constant<int, 8 + j>{}), acc[i][j], 0, 0, 0);
  };
  // the reads of a step in the order its MFMAs first use them (A0, B0..B7,
  // A1..A7), one instruction after each MFMA: a transposed fragment takes two
  using ReadOps = ReadSchedule<TA, TB>;
  constexpr int kPerStep = 2 * kJ;  // loads per wave per step
  constexpr int kMfmas = 64;        // MFMAs per wave per step
  constexpr int kSpread = kMfmas / kPerStep;
  // The loads of a step are issued evenly over the MFMAs that follow its
  // fragment reads, except in the dL/dh product (only B transposed), which
  // keeps one load per kSpread MFMAs from the start of the step: each was
  // the faster order for its product (a load issued in the same slots as the
  // reads holds the wave's MFMA issue back longer).
  constexpr bool kLoadsAfterReads = TA || !TB;
  using I0 = std::integral_constant<int, 0>;

  const int nk = K / kBK;
  const int last = nk > 0 ? nk - 1 : 0;
  static_for<kStages>([&](auto st) { load_step(min((int)st.value, last), st.value); });
  __builtin_amdgcn_s_waitcnt(wait_vm((kStages - 1) * kPerStep));  // step 0 has landed
  __builtin_amdgcn_s_barrier();
  static_for<16>([&](auto q) { fread(I0{}, I0{}, q, std::integral_constant<int, -1>{}); });
  __builtin_amdgcn_s_waitcnt(wait_vm((kStages - 2) * kPerStep));  // step 1 has landed
  __builtin_amdgcn_s_barrier();  // and every wave holds step 0: its stage is free

  // step kt (in LDS stage st) from register set `cur`; reads step kt+1 into
  // the other set; loads step kt+5 into the stage of step kt (free since the
  // last barrier)
  auto step = [&](int kt, auto cur, auto st) {
    using Nxt = std::integral_constant<int, cur.value ^ 1>;
    using StNxt = std::integral_constant<int, (st.value + 1) % kStages>;
    const int nkt = min(kt + kStages, last);
    char* nl = smem + st.value * kStage + w * 1024;
    static_for<kMfmas>([&](auto m) {
      mfma(cur, m);
      if constexpr (m.value < ReadOps::kOps)
        fread(Nxt{}, StNxt{}, std::integral_constant<int, ReadOps::q(m.value)>{},
              std::integral_constant<int, ReadOps::part(m.value)>{});
      if constexpr (kLoadsAfterReads) {
        constexpr int l0 = ReadOps::kOps, ls = (kMfmas - l0) / kPerStep;
        if constexpr (m.value >= l0 && (m.value - l0) % ls == 0 && (m.value - l0) / ls < kPerStep)
          load(nkt, nl, std::integral_constant<int, (m.value - l0) / ls>{});
      } else if constexpr (m.value % kSpread == kSpread - 1) {
        load(nkt, nl, std::integral_constant<int, m.value / kSpread>{});
      }
      __builtin_amdgcn_sched_barrier(0);
    });
    // reads of step kt+1 returned; this wave's loads of step kt+2 landed
    __builtin_amdgcn_s_waitcnt(wait_vm(3 * kPerStep));
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
  };
  // unrolled over both register sets and the ring: every stage is a constant
  // (an epilogue whose K is never empty lets the compiler drop the path that
  // reaches it with the zero-initialised accumulators, which otherwise holds
  // copies of them in registers across the loop)
  const int nk_loop = Epi::kKPositive ? max(nk, 1) : nk;
  for (int kt0 = 0; kt0 < nk_loop; kt0 += 2 * kStages)
    static_for<2 * kStages>([&](auto u) {
      if (kt0 + u.value < nk)
        step(kt0 + u.value, std::integral_constant<int, u.value % 2>{},
             std::integral_constant<int, u.value % kStages>{});
    });
  // every load (including the clamped ones past the last step) has landed
  // before the epilogue reuses LDS
  __builtin_amdgcn_s_waitcnt(wait_vm(0));
  __syncthreads();

  // The epilogue recomputes its indexes from an opaque copy of the lane id,
  // so that none of them is computed before the main loop and held in
  // registers across it.
  Frag fe = f;
  asm volatile("" : "+v"(fe.lane));
  epi(acc, fe, m_valid, n_valid, smem, pre);
}

void launch_gemm_lse(const GemmArgs& g, const int32_t* y_p, float* zy, float2* ms, int64_t ldms,
                     int64_t V, int64_t v0, hipStream_t s) {
  hipLaunchKernelGGL((k_gemm<EpiLse, false, false>), dim3(gemm_grid(g.tiles_m, g.tiles_n)),
                     dim3(256), 0, s, g, EpiLse{y_p, zy, ms, ldms, V, v0});
}

void launch_gemm_dz(const GemmArgs& g, const float* lse_p, const float* g_p, uint16_t* dz,
                    int64_t dz_kt, int64_t V, int64_t v0, hipStream_t s) {
  hipLaunchKernelGGL((k_gemm<EpiDz, false, false>), dim3(gemm_grid(g.tiles_m, g.tiles_n)),
                     dim3(256), 0, s, g, EpiDz{lse_p, g_p, dz, dz_kt, V, v0});
}

// Distinct kernel symbols (hence distinct entries in profiles) for the two
// gradient products that share the store epilogue.
void launch_gemm_store(const GemmArgs& g, const StoreArgs& a, bool grad_weight, hipStream_t s) {
  const EpiStore e{a};
  const dim3 blocks(gemm_grid(g.tiles_m, g.tiles_n), g.splits > 1 ? g.splits : 1);
  if (grad_weight)
    hipLaunchKernelGGL((k_gemm<EpiGradWeight, true, true>), blocks, dim3(256), 0, s, g,
                       EpiGradWeight{e});
  else
    hipLaunchKernelGGL((k_gemm<EpiGradHidden, false, true>), blocks, dim3(256), 0, s, g,
                       EpiGradHidden{e});
}

}  // namespace grpo
