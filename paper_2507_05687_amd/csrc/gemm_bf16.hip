// bf16 MFMA contraction C[m, n] = sum_k A[m, k] * B[n, k] for gfx950, with
// fused epilogues for the three uses on the GRPO path:
//
//   EpiLse   forward scoring: A = LM-head rows (vocabulary), B = hidden rows
//            (tokens). Reduces each token column of the 256x256 tile to an
//            online (max, sum-exp) partial and picks out z at the sampled id.
//   EpiDz    backward: the same tile recomputed, turned into
//            dz = g * (1[v = y] - exp(z - lse)) and stored in bf16 both
//            token-major and vocabulary-major.
//   EpiStore dL/dh = dz . W and dL/dW = dz^T . h: fp32 stores, optionally
//            accumulating, gathering output rows, or converting to bf16.
//
// Tiling: one 512-thread workgroup per 256x256 output tile, K in steps of
// 32 from operands in the library's tiled layout (see the main loop).
//
// Tile order: workgroup ids are dealt round-robin to the 8 XCDs, so id
// b runs on XCD b % 8. Tiles are assigned so that each XCD owns a band of
// kGM tile-rows and walks the tile-columns in blocks of kGN, and all 8 XCDs
// walk the same columns at the same time: the B operand is then shared
// through the last-level cache and each XCD's L2 sees only kGM + kGN
// distinct operand slices per K step. Products with fewer than 8 kGM
// tile-rows split the valid tile-columns among the XCDs instead. A product
// may also split K over the grid's y dimension (partial sums to a buffer).
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

// Maps a workgroup id to its (tile_m, tile_n); returns false for the
// padding workgroups of the last band. With fewer than 8 kGM tile-rows there
// are not enough rows for a band per XCD (column_tile_of).
__device__ inline bool tile_of(int bid, int tiles_m, int tiles_n, int& tm, int& tn) {
  int xcd = bid & 7, loc = bid >> 3;
  int per_band = kGM * tiles_n;
  int band = loc / per_band;
  int r = loc - band * per_band;
  int nb = r / (kGM * kGN);
  int r2 = r - nb * (kGM * kGN);
  tm = band * (8 * kGM) + xcd * kGM + r2 % kGM;
  tn = nb * kGN + r2 / kGM;
  return tm < tiles_m;
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

// Tile of this workgroup, or false if it has none (or only rows or columns
// past the valid counts). The mapping is chosen by the grid's tile-rows.
__device__ inline bool gemm_tile(const GemmArgs& g, int m_valid, int n_valid, int& tm, int& tn) {
  if (g.tiles_m < 8 * kGM) {
    if (m_valid <= 0 || n_valid <= 0) return false;
    return column_tile_of(blockIdx.x, min(g.tiles_m, (int)ceil_div(m_valid, kTile)),
                          min(g.tiles_n, (int)ceil_div(n_valid, kTile)), tm, tn);
  }
  return tile_of(blockIdx.x, g.tiles_m, g.tiles_n, tm, tn) && tm * kTile < m_valid &&
         tn * kTile < n_valid;
}

int gemm_grid(int tiles_m, int tiles_n) {
  if (tiles_m < 8 * kGM) return 8 * tiles_m * (int)ceil_div(tiles_n, 8);
  return (int)ceil_div(tiles_m, 8 * kGM) * 8 * kGM * tiles_n;
}

// ------------------------------------------------------------ epilogues
struct Frag {
  int tm, tn, wm, wn, lane;
  int cbase;  // first tile column of this wave (wn * wave width)
  // row (within the 256x256 tile) of accumulator register r of block mi
  __device__ int row(int mi, int r) const {
    return wm * 128 + mi * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
  }
  __device__ int col(int ni) const { return cbase + ni * 32 + (lane & 31); }
};

struct EpiLse {
  const int32_t* y_p;  // sampled id of each packed token
  float* zy;           // z at the sampled id, per packed token
  float2* ms;          // [2 * tiles_m][ldms] partial (max, sum-exp) per 128-row half tile
  int64_t ldms;
  int64_t V;

  // Reduces this lane's 64 rows of column ni (rows with offset >= vlim are
  // past the vocabulary) to (max, sum exp(z - max)) and picks out z at y.
  template <bool FULL, int NI, class Acc>
  __device__ __forceinline__ void column(const Acc& acc, int ni, float& m_out, float& s_out,
                                         int vlim, int y, float* zy_t) const {
    float m = -INFINITY;
    static_for<4>([&](auto mi) {
      static_for<16>([&](auto r) {
        constexpr int o = mi * 32 + (r >> 2) * 8 + (r & 3);
        if (FULL || o < vlim) m = fmaxf(m, acc[mi][ni][r.value]);
      });
    });
    float s = 0.f;
    const float m2l = m * kLog2e;
    static_for<4>([&](auto mi) {
      static_for<16>([&](auto r) {
        constexpr int o = mi * 32 + (r >> 2) * 8 + (r & 3);
        if (FULL || o < vlim) s += __builtin_amdgcn_exp2f(fmaf(acc[mi][ni][r.value], kLog2e, -m2l));
        if (o == y) *zy_t = acc[mi][ni][r.value];
      });
    });
    m_out = m;
    s_out = s;
  }

  // the sampled id of each of this lane's columns, loaded before the main
  // loop so that the loop hides its latency (the per-token arrays hold a
  // value for every column of the grid; those past the valid tokens are
  // ignored)
  template <int NI>
  struct Pre {
    int y[NI];
  };
  template <int NI>
  __device__ __forceinline__ Pre<NI> prefetch(const Frag& f, int) const {
    Pre<NI> p;
    static_for<NI>([&](auto ni) { p.y[ni] = y_p[(int64_t)f.tn * kTile + f.col(ni)]; });
    return p;
  }

  template <int NI>
  __device__ __forceinline__ void operator()(f32x16 (&acc)[4][NI], const Frag& f, int m_valid,
                                             int n_valid, char*, const Pre<NI>& pre) const {
    const int vbase = f.tm * kTile + f.wm * 128 + (f.lane >> 5) * 4;
    const int vlim = (int)(V - vbase);  // rows r of this lane are valid iff row offset < vlim
    const bool full = (int64_t)f.tm * kTile + f.wm * 128 + 128 <= V;  // wave-uniform
    static_for<NI>([&](auto ni) {
      const int64_t t = (int64_t)f.tn * kTile + f.col(ni);
      const int y = t < n_valid ? pre.y[ni] - vbase : -1;  // y as a row offset of this lane
      float m, s;
      if (full)
        column<true, NI>(acc, ni, m, s, vlim, y, zy + t);
      else
        column<false, NI>(acc, ni, m, s, vlim, y, zy + t);
      // merge with the lane holding the other 64 rows of this column; each
      // 128-row half tile (wave row wm) writes its own partial
      float m2 = __shfl_xor(m, 32, 64), s2 = __shfl_xor(s, 32, 64);
      float mm = fmaxf(m, m2);
      float sm = (s == 0.f ? 0.f : s * __expf(m - mm)) + (s2 == 0.f ? 0.f : s2 * __expf(m2 - mm));
      if (f.lane < 32 && t < n_valid)
        ms[(int64_t)(2 * f.tm + f.wm) * ldms + t] = make_float2(mm, sm);
    });
  }
};

struct EpiDz {
  const int32_t* y_p;
  const float* lse_p;
  const float* g_p;
  uint16_t* dz;    // tiled [tokens][chunk vocabulary], dz_kt 32-wide blocks per tile-row
  int64_t dz_kt;
  uint16_t* dzT;   // tiled [chunk vocabulary][tokens] (may be NULL), dzT_kt blocks per tile-row
  int64_t dzT_kt;
  int64_t V;       // vocabulary size
  int64_t v0;      // first vocabulary row of this chunk

  // per column of this lane: sampled id, lse and g, loaded before the main
  // loop so that the loop hides their latency (the per-token arrays hold a
  // value for every column of the grid; those past the valid tokens are
  // ignored)
  template <int NI>
  struct Pre {
    int y[NI];
    float lse[NI], g[NI];
  };
  template <int NI>
  __device__ __forceinline__ Pre<NI> prefetch(const Frag& f, int) const {
    Pre<NI> p;
    static_for<NI>([&](auto ni) {
      const int64_t t = (int64_t)f.tn * kTile + f.col(ni);
      p.y[ni] = y_p[t];
      p.lse[ni] = lse_p[t];
      p.g[ni] = g_p[t];
    });
    return p;
  }

  template <int NI>
  __device__ __forceinline__ void operator()(f32x16 (&acc)[4][NI], const Frag& f, int m_valid,
                                             int n_valid, char* smem, const Pre<NI>& pre) const {
    const int hi = (f.lane >> 5) * 4;
    const int64_t vbase = v0 + (int64_t)f.tm * kTile + f.wm * 128 + hi;
    const int vlim = (int)((V - vbase) < (1 << 20) ? (V - vbase) : (1 << 20));
    // every row of this wave is inside the vocabulary: no per-element bound
    const bool full = v0 + (int64_t)f.tm * kTile + f.wm * 128 + 128 <= V;  // wave-uniform
    // this wave's staging area: its 128 x (32 NI) part of the tile as four
    // 32-wide vocabulary blocks of 32 NI token rows (64 bytes each)
    char* stage = smem + (f.wn * 2 + f.wm) * (NI * 8192);
    if (full)
      body(acc, f, pre, n_valid, vbase, vlim, stage, std::true_type{});
    else
      body(acc, f, pre, n_valid, vbase, vlim, stage, std::false_type{});
    // The LDS operations of one wave complete in order; the wait only makes
    // the staged values visible before any lane reads another lane's.
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
    const int64_t t0 = (int64_t)f.tn * kTile + f.cbase;  // the wave's first token
    // Token-major dz: the wave's part of each vocabulary block is 32 NI
    // consecutive 64-byte rows of one tiled block, written 16 bytes per lane
    // in whole lines.
    static_for<4>([&](auto mi) {
      uint16_t* pb = dz + ((t0 >> 8) * dz_kt + f.tm * 8 + f.wm * 4 + mi) * kTileElems;
      static_for<2 * NI>([&](auto it) {
        const int tl = it * 16 + (f.lane >> 2), c = f.lane & 3;
        const u32x4 v = *(const u32x4*)(stage + mi * (NI * 2048) + tl * 64 + (stage_chunk(tl, c) << 4));
        *(u32x4*)(pb + ((t0 & 255) + tl) * 32 + c * 8) = v;
      });
    });
    if (dzT == nullptr) return;
    // Vocabulary-major dzT: transposing LDS reads (ds_read_b64_tr_b16: within
    // each 16 lanes, lane i receives element i%4 of lanes i/4, 4 + i/4,
    // 8 + i/4, 12 + i/4) give each lane 8 consecutive tokens of one vocabulary
    // row; one store covers 16 rows x 32 tokens of a tiled block, 1 KiB.
    const int g4 = f.lane >> 4, i16 = f.lane & 15;
    const int jr = (f.lane >> 2) & 3, qv = f.lane & 3;  // source row / vocabulary quad
    static_for<NI>([&](auto ni) {
      uint16_t* pbt = dzT + ((int64_t)f.tm * dzT_kt + ((t0 >> 5) + ni)) * kTileElems +
                      (f.wm * 128) * 32;
      static_for<4>([&](auto mi) {
        static_for<2>([&](auto vh) {
          i16x4 r[2];
          static_for<2>([&](auto h) {
            const int tl = ni * 32 + g4 * 8 + h * 4 + jr;
            const int vq = vh * 16 + qv * 4;  // first of the 4 vocabulary entries read
            r[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (lds_i16x4_ptr_t)(stage + mi * (NI * 2048) + tl * 64 +
                                  (stage_chunk(tl, vq >> 3) << 4) + (vq & 7) * 2));
          });
          const u32x4 v = {__builtin_bit_cast(uint32_t, __builtin_shufflevector(r[0], r[0], 0, 1)),
                           __builtin_bit_cast(uint32_t, __builtin_shufflevector(r[0], r[0], 2, 3)),
                           __builtin_bit_cast(uint32_t, __builtin_shufflevector(r[1], r[1], 0, 1)),
                           __builtin_bit_cast(uint32_t, __builtin_shufflevector(r[1], r[1], 2, 3))};
          *(u32x4*)(pbt + (mi * 32 + vh * 16 + i16) * 32 + g4 * 8) = v;
        });
      });
    });
  }

  // Physical 16-byte chunk of logical chunk c in staging row tl: a row-dependent
  // XOR that keeps the staging writes at two lanes per bank and both readbacks
  // (16-byte row reads and transposing reads of four consecutive rows) free of
  // bank conflicts.
  static __device__ __forceinline__ int stage_chunk(int tl, int c) {
    const int m = (tl >> 1) & 3;
    return c ^ m ^ ((m & 1) << 1);
  }

  // dz of this lane's columns, in bf16, staged in LDS (token-major)
  template <int NI, class Full>
  __device__ __forceinline__ void body(f32x16 (&acc)[4][NI], const Frag& f, const Pre<NI>& pre,
                                       int n_valid, int64_t vbase, int vlim, char* stage,
                                       Full) const {
    const int hi = (f.lane >> 5) * 4;
    static_for<NI>([&](auto ni) {
      const int64_t t = (int64_t)f.tn * kTile + f.col(ni);
      const bool tv = t < n_valid;
      const int y = tv ? (int)(pre.y[ni] - vbase) : -1;  // y as a row offset of this lane
      // p = exp(z - lse) = exp2(z*log2e - lse*log2e); invalid columns get g = 0
      const float l2 = tv ? pre.lse[ni] * kLog2e : 0.f;
      const float g = tv ? pre.g[ni] : 0.f;
      const int tl = ni * 32 + (f.lane & 31);  // this column's row in the staging blocks
      static_for<4>([&](auto mi) {
        static_for<4>([&](auto q) {
          float d[4];
          static_for<4>([&](auto e) {
            constexpr int r = q * 4 + e;
            constexpr int o = mi * 32 + q * 8 + e;
            const float p = __builtin_amdgcn_exp2f(fmaf(acc[mi][ni][r], kLog2e, -l2));
            const float dv = g * (0.f - p);  // the sampled id's entry is redone below
            d[e] = (Full::value || o < vlim) ? dv : 0.f;
          });
          const uint32_t w0 = bf16_pack2(d[0], d[1]), w1 = bf16_pack2(d[2], d[3]);
          *(uint2*)(stage + mi * (NI * 2048) + tl * 64 + (stage_chunk(tl, q) << 4) + hi * 2) =
              make_uint2(w0, w1);
        });
      });
      // dz at the sampled id: g * (1 - p), written over its staged entry by
      // the one lane that holds it (row offsets o < 128 with o & 4 == 0)
      if ((unsigned)y < 128u && (y & 4) == 0) {
        static_for<4>([&](auto mi) {
          static_for<16>([&](auto r) {
            constexpr int q = r / 4, e = r % 4;
            constexpr int o = mi * 32 + q * 8 + e;
            if (o == y) {
              const float p = __builtin_amdgcn_exp2f(fmaf(acc[mi][ni][r.value], kLog2e, -l2));
              *(uint16_t*)(stage + mi * (NI * 2048) + tl * 64 + (stage_chunk(tl, q) << 4) +
                           hi * 2 + e * 2) = bf16_bits(g * (1.f - p));
            }
          });
        });
      }
    });
  }
};

struct EpiStore {
  float* acc_buf;        // fp32 accumulation buffer; every row/column of every tile exists
  int64_t ld_acc;
  int read_acc;          // add the buffer's current value
  void* out;             // final output (NULL: write acc_buf instead)
  int64_t ld_out;
  int out_bf16;
  int add_out;           // add the output's current value (fp32 output only)
  const int32_t* out_rows;  // output row = out_rows[m] (NULL: m)
  int64_t m_limit;       // rows >= m_limit are not stored (static bound)
  int64_t n_limit;       // columns >= n_limit are not stored
  int64_t split_stride;  // with a split K, split y writes acc_buf + y * split_stride

  template <int NI>
  struct Pre {};
  template <int NI>
  __device__ __forceinline__ Pre<NI> prefetch(const Frag&, int) const {
    return {};
  }

  template <int NI>
  __device__ __forceinline__ void operator()(f32x16 (&acc)[4][NI], const Frag& f, int m_valid,
                                             int n_valid, char*, const Pre<NI>&) const {
    const int64_t mlim = m_limit < m_valid ? m_limit : m_valid;
    const int64_t m0 = (int64_t)f.tm * kTile + f.wm * 128 + (f.lane >> 5) * 4;
    const int64_t n0 = (int64_t)f.tn * kTile + f.cbase + (f.lane & 31);
    const bool full = (int64_t)f.tm * kTile + kTile <= mlim &&
                      (int64_t)f.tn * kTile + kTile <= n_limit;
    float* pacc = acc_buf ? acc_buf + blockIdx.y * split_stride + m0 * ld_acc + n0 : nullptr;
    // Batches of RB rows x NI columns of this lane (16 or 32 values): each
    // batch is loaded, combined and stored before the next starts, so the
    // loads of a batch are in flight together and its registers die right
    // after. (mi, r) -> row offset mi*32 + (r/4)*8 + r%4; ni -> column ni*32.
    constexpr int RB = NI >= 4 ? 4 : 8;
    constexpr int kPerMi = 16 / RB;
    static_for<4 * kPerMi>([&](auto bq) {
      constexpr int mi = bq / kPerMi, r0 = (bq % kPerMi) * RB;
      float v[RB][NI];
      static_for<RB>([&](auto rr) {
        static_for<NI>([&](auto ni) { v[rr][ni] = acc[mi][ni][r0 + rr]; });
      });
      if (read_acc) {  // the accumulation buffer holds every row/column of the tile
        float prev[RB][NI];
        static_for<RB>([&](auto rr) {
          constexpr int r = r0 + rr;
          constexpr int o = mi * 32 + (r >> 2) * 8 + (r & 3);
          const float* pr = pacc + o * ld_acc;
          static_for<NI>([&](auto ni) { prev[rr][ni] = pr[ni * 32]; });
        });
        static_for<RB>([&](auto rr) {
          static_for<NI>([&](auto ni) { v[rr][ni] += prev[rr][ni]; });
        });
      }
      if (out == nullptr) {
        static_for<RB>([&](auto rr) {
          constexpr int r = r0 + rr;
          constexpr int o = mi * 32 + (r >> 2) * 8 + (r & 3);
          float* pr = pacc + o * ld_acc;
          static_for<NI>([&](auto ni) { pr[ni * 32] = v[rr][ni]; });
        });
      } else if (full) {
        int64_t orow[RB];
        static_for<RB>([&](auto rr) {
          constexpr int r = r0 + rr;
          constexpr int o = mi * 32 + (r >> 2) * 8 + (r & 3);
          orow[rr] = (out_rows ? (int64_t)out_rows[m0 + o] : m0 + o) * ld_out + n0;
        });
        if (out_bf16) {
          uint16_t* ob = (uint16_t*)out;
          static_for<RB>([&](auto rr) {
            static_for<NI>([&](auto ni) { ob[orow[rr] + ni * 32] = bf16_bits(v[rr][ni]); });
          });
        } else {
          float* of = (float*)out;
          if (add_out) {
            float prev[RB][NI];
            static_for<RB>([&](auto rr) {
              static_for<NI>([&](auto ni) { prev[rr][ni] = of[orow[rr] + ni * 32]; });
            });
            static_for<RB>([&](auto rr) {
              static_for<NI>([&](auto ni) { v[rr][ni] += prev[rr][ni]; });
            });
          }
          static_for<RB>([&](auto rr) {
            static_for<NI>([&](auto ni) { of[orow[rr] + ni * 32] = v[rr][ni]; });
          });
        }
      } else {  // edge tile: per-element bounds
        static_for<RB>([&](auto rr) {
          constexpr int r = r0 + rr;
          constexpr int o = mi * 32 + (r >> 2) * 8 + (r & 3);
          const int64_t m = m0 + o;
          if (m < mlim) {
            const int64_t orow = out_rows ? (int64_t)out_rows[m] : m;
            static_for<NI>([&](auto ni) {
              const int64_t n = n0 + ni * 32;
              if (n < n_limit) {
                if (out_bf16) {
                  ((uint16_t*)out)[orow * ld_out + n] = bf16_bits(v[rr][ni]);
                } else {
                  float* o2 = (float*)out + orow * ld_out + n;
                  *o2 = add_out ? *o2 + v[rr][ni] : v[rr][ni];
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

// Distinct types (hence distinct kernel symbols in profiles) for the two
// gradient products that share the store epilogue.
struct EpiGradHidden : EpiStore {};
struct EpiGradWeight : EpiStore {};

// ------------------------------------------------------------ main loop
// Both operands are in the tiled layout: tile-row r of an operand is a run
// of 256 x 32 blocks (16 KiB each, rows of 64 bytes), block kb of it at
// (r * kt + kb0 + kb) * 8192 elements. One K step (32) of a tile is then
// one contiguous 16 KiB block per operand, and each 1 KiB load instruction
// of a wave covers eight whole 128-byte lines.
//
// Eight waves of 64 (two per SIMD); wave w owns rows (w%2)*128 and columns
// (w/2)*64 of the tile as 4 x 2 blocks of 32x32x16 MFMAs (128 fp32
// accumulators per lane), so that one wave's MFMAs can run while the other
// wave of its SIMD waits on LDS, a load or a barrier.
//
// LDS is a ring of 5 stages of 32 KiB (A block + B block of one K step).
// After the barrier of step kt every wave has read step kt, so its stage
// receives step kt+5; those four loads per wave are spread over the MFMAs
// up to the next barrier (one per four MFMAs), which keeps the load
// pipeline fed without stalling MFMA issue on a full load queue, and each
// step is requested about four steps before it is read.
constexpr int kWaves = 8;
constexpr int kWN = 64;                    // columns per wave
constexpr int kNI = kWN / 32;              // MFMA blocks per wave along N
constexpr int kStage = 2 * kTileElems * 2; // bytes of one A + B stage
constexpr int kStages = 5;
constexpr int kJ = kTileElems * 2 / 1024 / kWaves;  // 1 KiB loads per operand per wave per step

template <class Epi>
__global__ void __launch_bounds__(64 * kWaves, 1) k_gemm_bf16(GemmArgs g, Epi epi) {
  constexpr int NI = kNI;
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
  const Frag f{tm, tn, wm, wn, lane, wn * kWN};
  const auto pre = epi.template prefetch<NI>(f, n_valid);

  f32x16 acc[4][NI];
  static_for<4>([&](auto i) {
    static_for<NI>([&](auto j) {
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    });
  });

  // ---- loads: the j-th load of lane l of wave w fills stage row
  // q = 16*(w + 8j) + l/4 at physical chunk l%4, i.e. logical chunk
  // (l%4) ^ ((q/4)%4); one instruction writes 1 KiB of consecutive LDS.
  const int qrow = 16 * w + (lane >> 2);
  const int qch = (lane & 3) ^ ((qrow >> 2) & 3);  // the same for q + 128j
  // load l of step kt (l < kJ: A part l, else B part l - kJ) into stage bytes la
  const __amdgpu_buffer_rsrc_t ra =
      tile_rsrc(g.A + ((int64_t)tm * g.a_kt + g.a_kb0 + kb0) * kTileElems);
  const __amdgpu_buffer_rsrc_t rb =
      tile_rsrc(g.B + ((int64_t)tn * g.b_kt + g.b_kb0 + kb0) * kTileElems);
  const uint32_t lofs = (uint32_t)(qrow * 32 + qch * 8) * 2;
  auto load = [&](int kt, char* la, auto l) {
    const uint32_t so = (uint32_t)kt * (kTileElems * 2);
    if constexpr (l.value < kJ)
      load_lds16(ra, la + l.value * 1024 * kWaves, lofs + l.value * 16 * kWaves * 64, so);
    else
      load_lds16(rb, la + kTileElems * 2 + (l.value - kJ) * 1024 * kWaves,
                 lofs + (l.value - kJ) * 16 * kWaves * 64, so);
  };
  auto load_step = [&](int kt, int stage) {
    char* la = smem + stage * kStage + w * 1024;
    static_for<2 * kJ>([&](auto l) { load(kt, la, l); });
  };

  // ---- fragment reads: lane reads row l%32 of each 32-row block, logical
  // chunk 2t + l/32 for sub-step t (K 16t .. 16t+15)
  const int fr = lane & 31;
  const int rd_a = (wm * 128 + fr) * 64;
  const int rd_b = kTileElems * 2 + (wn * kWN + fr) * 64;
  int rd_ch[2];
  static_for<2>([&](auto t) { rd_ch[t] = ((2 * t + (lane >> 5)) ^ ((fr >> 2) & 3)) << 4; });
  bf16x8 fa[2][4], fb[2][NI];
  // fragment r (A blocks first, then B blocks) of sub-step t of step kt
  // fragment r (A blocks first, then B blocks) of sub-step t from LDS stage st
  auto fread = [&](auto slot, auto st, int t, auto r) {
    const char* base = smem + st.value * kStage;
    if constexpr (r.value < 4)
      fa[slot.value][r.value] = *(const bf16x8*)(base + rd_a + r.value * 32 * 64 + rd_ch[t]);
    else
      fb[slot.value][r.value - 4] =
          *(const bf16x8*)(base + rd_b + (r.value - 4) * 32 * 64 + rd_ch[t]);
  };
  constexpr int kReads = 4 + NI;  // fragment reads per sub-step
  auto fread_half = [&](auto slot, auto st, int t, auto h) {
    static_for<kReads>([&](auto r) {
      if constexpr ((r.value < kReads / 2) == (h.value == 0)) fread(slot, st, t, r);
    });
  };
  auto mfma = [&](auto slot, auto m) {
    constexpr int i = m.value / NI, j = m.value % NI;
    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[slot.value][i], fb[slot.value][j],
                                                        acc[i][j], 0, 0, 0);
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  constexpr int kMfmas = 4 * NI;                  // MFMAs per sub-step
  constexpr int kSpread = kMfmas / kJ;            // MFMAs per load
  constexpr int kPerStep = 2 * kJ;                // loads per wave per step

  const int nk = K / kBK;
  const int last = nk > 0 ? nk - 1 : 0;  // K = 0 (no valid tokens) still loads step 0
  static_for<kStages>([&](auto st) { load_step(min((int)st.value, last), st.value); });
  __builtin_amdgcn_s_waitcnt(wait_vm((kStages - 1) * kPerStep));  // step 0 has landed
  __builtin_amdgcn_s_barrier();
  fread_half(I0{}, I0{}, 0, I0{});
  fread_half(I0{}, I0{}, 0, I1{});

  // The instruction order is fixed by scheduling fences. Each sub-step's
  // MFMAs run on fragments read one sub-step earlier; the next sub-step's
  // reads go out right after its first two MFMAs. Step kt: sub-step 0 (with
  // the B half of step kt+4's loads), wait for step kt+1, barrier, sub-step
  // 1 (with the A half of step kt+5's loads and the reads of step kt+1).
  // Past the end the last step is loaded again, into free stages only. The
  // loop is unrolled over the ring, so every LDS stage is a constant.
  auto step = [&](int kt, auto st) {
    constexpr int S = st.value;
    using Nxt = std::integral_constant<int, (S + 1) % kStages>;
    const int nkt_b = min(kt + kStages - 1, last);  // into the stage of step kt-1
    static_for<kMfmas>([&](auto m) {
      mfma(I0{}, m);
      if constexpr (m.value < 2) fread_half(I1{}, st, 1, std::integral_constant<int, m.value>{});
      if constexpr (m.value % kSpread == kSpread - 1) {
        if (kt > 0)
          load(nkt_b, smem + ((S + kStages - 1) % kStages) * kStage + w * 1024,
               std::integral_constant<int, kJ + m.value / kSpread>{});
      }
      __builtin_amdgcn_sched_barrier(0);
    });
    __builtin_amdgcn_s_waitcnt(wait_vm(3 * kPerStep));  // step kt+1 has landed
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    const int nkt_a = min(kt + kStages, last);  // into the stage of step kt
    static_for<kMfmas>([&](auto m) {
      if constexpr (m.value % kSpread == kSpread - 1)
        load(nkt_a, smem + S * kStage + w * 1024, std::integral_constant<int, m.value / kSpread>{});
      mfma(I1{}, m);
      if constexpr (m.value == 1 || m.value == 2)
        fread_half(I0{}, Nxt{}, 0, std::integral_constant<int, m.value - 1>{});
      __builtin_amdgcn_sched_barrier(0);
    });
  };
  for (int kt0 = 0; kt0 < nk; kt0 += kStages)
    static_for<kStages>([&](auto st) {
      if (kt0 + st.value < nk) step(kt0 + st.value, st);
    });
  __syncthreads();  // every load has landed before LDS is reused

  epi(acc, f, m_valid, n_valid, smem, pre);
}

// ---- four-wave variant: one wave per SIMD, each owning 128x128 as 4x4
// blocks (256 fp32 accumulators per lane, in AGPRs). A wave reads the
// fragments of a whole K step (both 16-wide sub-steps, 64 VGPRs) into
// registers one step ahead, so its MFMAs never wait on LDS; the barrier at
// the end of step kt (after every wave's reads of step kt+1 have returned
// and its loads of step kt+2 have landed) frees the stage of step kt+1 for
// the loads of step kt+6. Eight waves of 128x64 read 1.5x the LDS bytes per
// flop of this layout.
constexpr int kW4Waves = 4;
constexpr int kW4J = kTileElems * 2 / 1024 / kW4Waves;  // 1 KiB loads per operand per wave per step

template <class Epi>
__global__ void __launch_bounds__(64 * kW4Waves, 1) k_gemm_w4(GemmArgs g, Epi epi) {
  constexpr int NI = 4;
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
  const Frag f{tm, tn, wm, wn, lane, wn * 128};
  const auto pre = epi.template prefetch<NI>(f, n_valid);

  f32x16 acc[4][NI];
  static_for<4>([&](auto i) {
    static_for<NI>([&](auto j) {
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    });
  });

  const int qrow = 16 * w + (lane >> 2);
  const int qch = (lane & 3) ^ ((qrow >> 2) & 3);
  const __amdgpu_buffer_rsrc_t ra =
      tile_rsrc(g.A + ((int64_t)tm * g.a_kt + g.a_kb0 + kb0) * kTileElems);
  const __amdgpu_buffer_rsrc_t rb =
      tile_rsrc(g.B + ((int64_t)tn * g.b_kt + g.b_kb0 + kb0) * kTileElems);
  const uint32_t lofs = (uint32_t)(qrow * 32 + qch * 8) * 2;
  // load l of step kt (l < kW4J: A part l, else B part l - kW4J) into stage bytes la
  auto load = [&](int kt, char* la, auto l) {
    const uint32_t so = (uint32_t)kt * (kTileElems * 2);
    if constexpr (l.value < kW4J)
      load_lds16(ra, la + l.value * 1024 * kW4Waves, lofs + l.value * 16 * kW4Waves * 64, so);
    else
      load_lds16(rb, la + kTileElems * 2 + (l.value - kW4J) * 1024 * kW4Waves,
                 lofs + (l.value - kW4J) * 16 * kW4Waves * 64, so);
  };
  auto load_step = [&](int kt, int stage) {
    char* la = smem + stage * kStage + w * 1024;
    static_for<2 * kW4J>([&](auto l) { load(kt, la, l); });
  };

  const int fr = lane & 31;
  const int rd_a = (wm * 128 + fr) * 64;
  const int rd_b = kTileElems * 2 + (wn * 128 + fr) * 64;
  int rd_ch[2];
  static_for<2>([&](auto t) { rd_ch[t] = ((2 * t + (lane >> 5)) ^ ((fr >> 2) & 3)) << 4; });
  // fragments of one step: q = t*8 + r, r < 4 A block r, else B block r-4
  bf16x8 fs[2][16];
  // fragment q of a step from LDS stage st
  auto fread = [&](auto slot, auto st, auto q) {
    constexpr int t = q.value / 8, r = q.value % 8;
    const char* base = smem + st.value * kStage;
    if constexpr (r < 4)
      fs[slot.value][q.value] = *(const bf16x8*)(base + rd_a + r * 32 * 64 + rd_ch[t]);
    else
      fs[slot.value][q.value] = *(const bf16x8*)(base + rd_b + (r - 4) * 32 * 64 + rd_ch[t]);
  };
  // MFMA m of a step: sub-step t = m/16, A block i, B block j
  auto mfma = [&](auto slot, auto m) {
    constexpr int t = m.value / 16, i = (m.value / 4) % 4, j = m.value % 4;
    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fs[slot.value][t * 8 + i],
                                                        fs[slot.value][t * 8 + 4 + j], acc[i][j],
                                                        0, 0, 0);
  };
  constexpr int kPerStep = 2 * kW4J;   // loads per wave per step
  constexpr int kMfmas = 32;           // MFMAs per wave per step
  constexpr int kSpread = kMfmas / kPerStep;
  using I0 = std::integral_constant<int, 0>;

  const int nk = K / kBK;
  const int last = nk > 0 ? nk - 1 : 0;
  static_for<kStages>([&](auto st) { load_step(min((int)st.value, last), st.value); });
  __builtin_amdgcn_s_waitcnt(wait_vm((kStages - 1) * kPerStep));  // step 0 has landed
  __builtin_amdgcn_s_barrier();
  static_for<16>([&](auto q) { fread(I0{}, I0{}, q); });
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
      if constexpr (m.value < 16) fread(Nxt{}, StNxt{}, m);
      if constexpr (m.value % kSpread == kSpread - 1)
        load(nkt, nl, std::integral_constant<int, m.value / kSpread>{});
      __builtin_amdgcn_sched_barrier(0);
    });
    // reads of step kt+1 returned; this wave's loads of step kt+2 landed
    __builtin_amdgcn_s_waitcnt(wait_vm(3 * kPerStep));
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
  };
  // unrolled over both register sets and the ring: every stage is a constant
  for (int kt0 = 0; kt0 < nk; kt0 += 2 * kStages)
    static_for<2 * kStages>([&](auto u) {
      if (kt0 + u.value < nk)
        step(kt0 + u.value, std::integral_constant<int, u.value % 2>{},
             std::integral_constant<int, u.value % kStages>{});
    });
  __syncthreads();  // every load has landed before LDS is reused

  epi(acc, f, m_valid, n_valid, smem, pre);
}

// The two gradient products (long K, fp32 store epilogues) run faster on the
// four-wave loop; the scoring and dz products on the eight-wave one.
template <class Epi>
constexpr bool four_waves() {
  return std::is_same<Epi, EpiGradWeight>::value || std::is_same<Epi, EpiGradHidden>::value;
}

template <class Epi>
static void launch_gemm(const GemmArgs& g, const Epi& e, hipStream_t s) {
  int grid = gemm_grid(g.tiles_m, g.tiles_n);
  const dim3 blocks(grid, g.splits > 1 ? g.splits : 1);
  if constexpr (four_waves<Epi>())
    hipLaunchKernelGGL((k_gemm_w4<Epi>), blocks, dim3(64 * kW4Waves), 0, s, g, e);
  else
    hipLaunchKernelGGL((k_gemm_bf16<Epi>), blocks, dim3(64 * kWaves), 0, s, g, e);
}

void launch_gemm_lse(const GemmArgs& g, const int32_t* y_p, float* zy, float2* ms, int64_t ldms,
                     int64_t V, hipStream_t s) {
  EpiLse e{y_p, zy, ms, ldms, V};
  launch_gemm<EpiLse>(g, e, s);
}

void launch_gemm_dz(const GemmArgs& g, const int32_t* y_p, const float* lse_p, const float* g_p,
                    uint16_t* dz, int64_t dz_kt, uint16_t* dzT, int64_t dzT_kt, int64_t V,
                    int64_t v0, hipStream_t s) {
  EpiDz e{y_p, lse_p, g_p, dz, dz_kt, dzT, dzT_kt, V, v0};
  launch_gemm<EpiDz>(g, e, s);
}

void launch_gemm_store(const GemmArgs& g, const StoreArgs& a, bool grad_weight, hipStream_t s) {
  EpiStore e{a.acc_buf, a.ld_acc,   a.read_acc, a.out,     a.ld_out,      a.out_bf16,
             a.add_out, a.out_rows, a.m_limit,  a.n_limit, a.split_stride};
  if (grad_weight)
    launch_gemm<EpiGradWeight>(g, EpiGradWeight{e}, s);
  else
    launch_gemm<EpiGradHidden>(g, EpiGradHidden{e}, s);
}

}  // namespace grpo
