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
// Tiling: one 256-thread workgroup (4 waves of 64) per 256x256 output tile;
// each wave owns a 128x128 quarter as a 4x4 grid of 32x32x16 bf16 MFMA
// blocks (256 fp32 accumulators per lane). K advances 64 at a time through a
// double-buffered LDS stage of 2 x (256x64 A + 256x64 B) bf16 = 128 KiB.
// LDS rows are 128 bytes; the eight 16-byte chunks of a row are XOR-swizzled
// by a few row bits so that the MFMA fragment reads hit distinct banks.
//
// Operands come row-major (the caller's hidden states and LM head) or in the
// tiled layout that the library writes for its own intermediates: 256-row x
// 64-column blocks stored contiguously, block (rb, kb) at
// (rb * blocks_per_row + kb) * 16384 elements. A K step of a tile then reads
// one contiguous 32 KiB block per operand.
//
// Tile order: workgroup ids are dealt round-robin to the 8 XCDs, so id
// b runs on XCD b % 8. Tiles are assigned so that each XCD owns a band of
// kGM tile-rows and walks the tile-columns in blocks of kGN, and all 8 XCDs
// walk the same columns at the same time: the B operand is then shared
// through the last-level cache and each XCD's L2 sees only kGM + kGN
// distinct operand slices per K step.
#include "kernels.h"

namespace grpo {

constexpr int kGM = 4;  // tile-rows per XCD band
constexpr int kGN = 8;  // tile-columns per step of the walk
constexpr int kLdsStage = 2 * kTile * kBK * 2;  // bytes of one A+B stage (64 KiB)

#ifndef GRPO_SWZ_SHIFT
#define GRPO_SWZ_SHIFT 1
#endif

__device__ inline int swz(int row) { return (row >> GRPO_SWZ_SHIFT) & 7; }

// s_waitcnt immediate that waits for LDS/scalar-memory counters only
// (vmcnt and expcnt left at their maxima).
constexpr int kWaitLgkmOnly = 0xC07F;

typedef __attribute__((address_space(1))) void* glb_ptr_t;
typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Maps a workgroup id to its (tile_m, tile_n); returns false for the
// padding workgroups of the last band.
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

int gemm_grid(int tiles_m, int tiles_n) {
  int bands = (int)ceil_div(tiles_m, 8 * kGM);
  return bands * 8 * kGM * tiles_n;
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
  float2* ms;          // [tiles_m][ldms] partial (max, sum-exp)
  int64_t ldms;
  int64_t V;

  template <int NI>
  __device__ __forceinline__ void operator()(f32x16 (&acc)[4][NI], const Frag& f, int m_valid,
                                             int n_valid,
                             char* smem) const {
    float pm[NI], ps[NI];
    const int vbase = f.tm * kTile + f.wm * 128 + (f.lane >> 5) * 4;
    const int vlim = (int)(V - vbase);  // rows r of this lane are valid iff row offset < vlim
    static_for<NI>([&](auto ni) {
      const int64_t t = (int64_t)f.tn * kTile + f.col(ni);
      const int y = t < n_valid ? y_p[t] - vbase : -1;  // y as a row offset of this lane
      float m = -INFINITY;
      static_for<4>([&](auto mi) {
        static_for<16>([&](auto r) {
          constexpr int o = mi * 32 + (r >> 2) * 8 + (r & 3);
          if (o < vlim) m = fmaxf(m, acc[mi][ni][r.value]);
        });
      });
      float s = 0.f;
      const float m2l = m * kLog2e;
      static_for<4>([&](auto mi) {
        static_for<16>([&](auto r) {
          constexpr int o = mi * 32 + (r >> 2) * 8 + (r & 3);
          if (o < vlim) s += __builtin_amdgcn_exp2f(fmaf(acc[mi][ni][r.value], kLog2e, -m2l));
          if (o == y) zy[t] = acc[mi][ni][r.value];
        });
      });
      // merge with the lane holding the other 64 rows of this column
      float m2 = __shfl_xor(m, 32, 64), s2 = __shfl_xor(s, 32, 64);
      float mm = fmaxf(m, m2);
      float sm = (s == 0.f ? 0.f : s * __expf(m - mm)) + (s2 == 0.f ? 0.f : s2 * __expf(m2 - mm));
      pm[ni] = mm;
      ps[ni] = sm;
    });
    // merge the two waves that share these columns (wm = 0 and 1)
    float2* xch = (float2*)smem;  // [256 tile columns]
    if (f.wm == 1 && f.lane < 32) {
      static_for<NI>([&](auto ni) {
        xch[f.cbase + ni * 32 + f.lane] = make_float2(pm[ni], ps[ni]);
      });
    }
    __syncthreads();
    if (f.wm == 0 && f.lane < 32) {
      static_for<NI>([&](auto ni) {
        float2 o = xch[f.cbase + ni * 32 + f.lane];
        float mm = fmaxf(pm[ni], o.x);
        float sm = (ps[ni] == 0.f ? 0.f : ps[ni] * __expf(pm[ni] - mm)) +
                   (o.y == 0.f ? 0.f : o.y * __expf(o.x - mm));
        int64_t t = (int64_t)f.tn * kTile + f.col(ni);
        if (t < n_valid) ms[(int64_t)f.tm * ldms + t] = make_float2(mm, sm);
      });
    }
  }
};

struct EpiDz {
  const int32_t* y_p;
  const float* lse_p;
  const float* g_p;
  uint16_t* dz;    // tiled [tokens][chunk vocabulary], dz_kt 64-wide blocks per tile-row
  int64_t dz_kt;
  uint16_t* dzT;   // tiled [chunk vocabulary][tokens] (may be NULL), dzT_kt blocks per tile-row
  int64_t dzT_kt;
  int64_t V;       // vocabulary size
  int64_t v0;      // first vocabulary row of this chunk

  template <int NI>
  __device__ __forceinline__ void operator()(f32x16 (&acc)[4][NI], const Frag& f, int m_valid,
                                             int n_valid, char*) const {
    const int hi = (f.lane >> 5) * 4;
    const int64_t vbase = v0 + (int64_t)f.tm * kTile + f.wm * 128 + hi;
    const int vlim = (int)((V - vbase) < (1 << 20) ? (V - vbase) : (1 << 20));
    static_for<NI>([&](auto ni) {
      const int64_t t = (int64_t)f.tn * kTile + f.col(ni);
      const bool tv = t < n_valid;
      const int y = tv ? (int)(y_p[t] - vbase) : -1;  // y as a row offset of this lane
      // p = exp(z - lse) = exp2(z*log2e - lse*log2e); invalid columns get g = 0
      const float l2 = tv ? lse_p[t] * kLog2e : 0.f;
      const float g = tv ? g_p[t] : 0.f;
      // element (t, vl) of dz lives at tile (t/256, vl/64), row t%256, column vl%64
      uint16_t* pz = dz + ((t >> 8) * dz_kt + f.tm * 4 + f.wm * 2) * kTileElems + (t & 255) * 64 + hi;
      // element (vl, t) of dzT lives at tile (vl/256, t/64), row vl%256, column t%64
      uint16_t* pzt = dzT ? dzT + ((int64_t)f.tm * dzT_kt + (t >> 6)) * kTileElems + (t & 63) +
                                (f.wm * 128 + hi) * 64
                          : nullptr;
      static_for<4>([&](auto mi) {
        static_for<4>([&](auto q) {
          float d[4];
          static_for<4>([&](auto e) {
            constexpr int r = q * 4 + e;
            constexpr int o = mi * 32 + q * 8 + e;
            const float p = __builtin_amdgcn_exp2f(fmaf(acc[mi][ni][r], kLog2e, -l2));
            const float dv = g * ((o == y ? 1.f : 0.f) - p);
            d[e] = o < vlim ? dv : 0.f;
          });
          const uint32_t w0 = bf16_pack2(d[0], d[1]), w1 = bf16_pack2(d[2], d[3]);
          if (pzt) {
            constexpr int o = mi * 32 + q * 8;
            pzt[o * 64] = (uint16_t)w0;
            pzt[(o + 1) * 64] = (uint16_t)(w0 >> 16);
            pzt[(o + 2) * 64] = (uint16_t)w1;
            pzt[(o + 3) * 64] = (uint16_t)(w1 >> 16);
          }
          *(uint2*)(pz + (mi >> 1) * kTileElems + (mi & 1) * 32 + q * 8) = make_uint2(w0, w1);
        });
      });
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

  template <int NI>
  __device__ __forceinline__ void operator()(f32x16 (&acc)[4][NI], const Frag& f, int m_valid,
                                             int n_valid, char*) const {
    const int64_t mlim = m_limit < m_valid ? m_limit : m_valid;
    const int64_t m0 = (int64_t)f.tm * kTile + f.wm * 128 + (f.lane >> 5) * 4;
    const int64_t n0 = (int64_t)f.tn * kTile + f.cbase + (f.lane & 31);
    const bool full = (int64_t)f.tm * kTile + kTile <= mlim &&
                      (int64_t)f.tn * kTile + kTile <= n_limit;
    float* pacc = acc_buf ? acc_buf + m0 * ld_acc + n0 : nullptr;
    // Batches of 32 values (8 rows x 4 columns of this lane): each batch is
    // loaded, combined and stored before the next starts, so the loads of a
    // batch are in flight together and its registers die right after.
    // (mi, r) -> row offset mi*32 + (r/4)*8 + r%4; ni -> column offset ni*32.
    static_for<8>([&](auto bq) {
      constexpr int mi = bq / 2, r0 = (bq % 2) * 8;
      float v[8][NI];
      static_for<8>([&](auto rr) {
        static_for<NI>([&](auto ni) { v[rr][ni] = acc[mi][ni][r0 + rr]; });
      });
      if (read_acc) {  // the accumulation buffer holds every row/column of the tile
        float prev[8][NI];
        static_for<8>([&](auto rr) {
          constexpr int r = r0 + rr;
          constexpr int o = mi * 32 + (r >> 2) * 8 + (r & 3);
          const float* pr = pacc + o * ld_acc;
          static_for<NI>([&](auto ni) { prev[rr][ni] = pr[ni * 32]; });
        });
        static_for<8>([&](auto rr) {
          static_for<NI>([&](auto ni) { v[rr][ni] += prev[rr][ni]; });
        });
      }
      if (out == nullptr) {
        static_for<8>([&](auto rr) {
          constexpr int r = r0 + rr;
          constexpr int o = mi * 32 + (r >> 2) * 8 + (r & 3);
          float* pr = pacc + o * ld_acc;
          static_for<NI>([&](auto ni) { pr[ni * 32] = v[rr][ni]; });
        });
      } else if (full) {
        int64_t orow[8];
        static_for<8>([&](auto rr) {
          constexpr int r = r0 + rr;
          constexpr int o = mi * 32 + (r >> 2) * 8 + (r & 3);
          orow[rr] = (out_rows ? (int64_t)out_rows[m0 + o] : m0 + o) * ld_out + n0;
        });
        if (out_bf16) {
          uint16_t* ob = (uint16_t*)out;
          static_for<8>([&](auto rr) {
            static_for<NI>([&](auto ni) { ob[orow[rr] + ni * 32] = bf16_bits(v[rr][ni]); });
          });
        } else {
          float* of = (float*)out;
          if (add_out) {
            float prev[8][NI];
            static_for<8>([&](auto rr) {
              static_for<NI>([&](auto ni) { prev[rr][ni] = of[orow[rr] + ni * 32]; });
            });
            static_for<8>([&](auto rr) {
              static_for<NI>([&](auto ni) { v[rr][ni] += prev[rr][ni]; });
            });
          }
          static_for<8>([&](auto rr) {
            static_for<NI>([&](auto ni) { of[orow[rr] + ni * 32] = v[rr][ni]; });
          });
        }
      } else {  // edge tile: per-element bounds
        static_for<8>([&](auto rr) {
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
// TILED: both operands are in the tiled layout (256x64 blocks, one block
// per K step, contiguous); otherwise both are row-major with a row stride,
// and B rows may be gathered through b_rows.
//
// WN is the width of one wave's output block: 128 (4 waves, one per SIMD,
// 4x4 MFMA blocks and 256 accumulators each) or 64 (8 waves, two per SIMD,
// 4x2 blocks and 128 accumulators each, so that one wave's MFMAs can run
// while the other waits on LDS or a barrier).
template <class Epi, bool KTAIL, bool TILED, int WN>
__global__ void __launch_bounds__(64 * 2 * (kTile / WN), 1) k_gemm_bf16(GemmArgs g, Epi epi) {
  constexpr int NI = WN / 32;               // MFMA blocks per wave along N
  constexpr int kWaves = 2 * (kTile / WN);  // 4 or 8
  constexpr int kJ = 32 / kWaves;           // 1 KiB LDS loads per operand per wave per step
  // 8 waves: ring of 5 stages of K = 32 (5 x 32 KiB); 4 waves: 2 stages of K = 64
  constexpr int kSmem = kWaves == 8 && !KTAIL ? 5 * 2 * kTile * 64 : 2 * kLdsStage;
  __shared__ __attribute__((aligned(16))) char smem[kSmem];
  int tm, tn;
  if (!tile_of(blockIdx.x, g.tiles_m, g.tiles_n, tm, tn)) return;
  int m_valid = g.m_dev ? min(*g.m_dev, g.M) : g.M;
  int n_valid = g.n_dev ? min(*g.n_dev, g.N) : g.N;
  if (tm * kTile >= m_valid || tn * kTile >= n_valid) return;
  int K = g.k_dev ? (int)round_up(*g.k_dev, kBK) : g.K;

  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  // wave -> output block: rows wm*128, columns wn*WN. With 8 waves, waves w
  // and w+4 share a SIMD and belong to different groups (see below).
  const int wm = w & 1, wn = w >> 1;

  // ---- fragment reads: lane reads row (l%32) of each 32-row block, chunk 2s + l/32
  const int fr = lane & 31;
  const int rd_base_a = (wm * 128 + fr) * 128;
  const int rd_base_b = kTile * kBK * 2 + (wn * WN + fr) * 128;
  int rd_ch[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) rd_ch[s] = ((2 * s + (lane >> 5)) ^ swz(fr)) << 4;

  f32x16 acc[4][NI];
  static_for<4>([&](auto i) {
    static_for<NI>([&](auto j) {
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    });
  });

  bf16x8 fa[2][4], fb[2][NI];
  auto fload = [&](int slot, const char* base, int s) {
    static_for<4>([&](auto i) {
      fa[slot][i] = *(const bf16x8*)(base + rd_base_a + i * 32 * 128 + rd_ch[s]);
    });
    static_for<NI>([&](auto i) {
      fb[slot][i] = *(const bf16x8*)(base + rd_base_b + i * 32 * 128 + rd_ch[s]);
    });
  };
  auto mfma_sub = [&](int slot) {
    static_for<4>([&](auto i) {
      static_for<NI>([&](auto j) {
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[slot][i], fb[slot][j], acc[i][j],
                                                            0, 0, 0);
      });
    });
  };
  constexpr int kMfma = 0x008, kVmem = 0x010, kDsRead = 0x100;
  constexpr int kSubMfma = 4 * NI, kSubReads = 4 + NI;
  // K step kt reads at +kt*64 (row-major) or +kt*kTileElems (tiled)
  constexpr int kStep = TILED ? kTileElems : kBK;

  if constexpr (!KTAIL) {
    // ---- global -> LDS directly (no register staging). The j-th load of
    // lane l of wave w fills LDS row r = 8*(w + kWaves*j) + l/8 at physical
    // chunk l%8, i.e. logical chunk (l%8) ^ swz(r); one load instruction of
    // a wave writes 1 KiB of consecutive LDS.
    const int drow = 8 * w + (lane >> 3);
    const int dch = (lane & 7) ^ swz(drow);  // swz(drow + 8*kWaves*j) == swz(drow)
    const uint16_t* sa[kJ];
    const uint16_t* sb[kJ];
    if (TILED) {
      const uint16_t* a0 =
          g.A + ((int64_t)tm * g.a_kt + g.a_kb0) * kTileElems + drow * 64 + dch * 8;
      const uint16_t* b0 =
          g.B + ((int64_t)tn * g.b_kt + g.b_kb0) * kTileElems + drow * 64 + dch * 8;
#pragma unroll
      for (int j = 0; j < kJ; ++j) {
        sa[j] = a0 + j * (8 * kWaves * 64);
        sb[j] = b0 + j * (8 * kWaves * 64);
      }
    } else {
#pragma unroll
      for (int j = 0; j < kJ; ++j) {
        int ra = min(tm * kTile + drow + 8 * kWaves * j, m_valid - 1);
        sa[j] = g.A + (int64_t)ra * g.lda + dch * 8;
        int rb = min(tn * kTile + drow + 8 * kWaves * j, n_valid - 1);
        if (g.b_rows) rb = g.b_rows[rb];
        sb[j] = g.B + (int64_t)rb * g.ldb + dch * 8;
      }
    }
    auto dma = [&](int kt, int buf) {
      const int64_t off = (int64_t)kt * kStep;
      char* la = smem + buf * kLdsStage + w * 1024;
      static_for<kJ>([&](auto j) {
        __builtin_amdgcn_global_load_lds((glb_ptr_t)(sa[j] + off),
                                         (lds_ptr_t)(la + j * 1024 * kWaves), 16, 0, 0);
      });
      static_for<kJ>([&](auto j) {
        __builtin_amdgcn_global_load_lds((glb_ptr_t)(sb[j] + off),
                                         (lds_ptr_t)(la + kTile * kBK * 2 + j * 1024 * kWaves),
                                         16, 0, 0);
      });
    };
      if constexpr (kWaves == 8) {
        // ---- 8 waves: K moves 32 at a time through a ring of 5 LDS stages
        // of 32 KiB (256 rows x 64 bytes for A and for B; the four 16-byte
        // chunks of a row are swizzled by (row/4)%4). Loads run 3 steps
        // ahead, so about three stages of data are in flight per CU, which
        // is what the L2-miss latency needs. Step kt: read sub-step 1, MFMAs
        // of sub-step 0; barrier (this thread's loads of step kt+1 have
        // landed -- steps kt+2 and kt+3 may still be in flight -- and every
        // read of stage kt is done); loads of step kt+4 into the stage step
        // kt-1 used; read sub-step 0 of step kt+1; MFMAs of sub-step 1.
        constexpr int kStage32 = 2 * kTile * 64;
        constexpr int kJ32 = 2;  // 1 KiB loads per operand per wave per step
        const int qrow = 16 * w + (lane >> 2);
        const int qch = (lane & 3) ^ ((qrow >> 2) & 3);  // same for row + 128j
        const uint16_t* qa[kJ32];
        const uint16_t* qb[kJ32];
        if (TILED) {
          const uint16_t* a0 =
              g.A + ((int64_t)tm * g.a_kt + g.a_kb0) * kTileElems + qrow * 64 + qch * 8;
          const uint16_t* b0 =
              g.B + ((int64_t)tn * g.b_kt + g.b_kb0) * kTileElems + qrow * 64 + qch * 8;
          static_for<kJ32>([&](auto j) {
            qa[j] = a0 + j * 128 * 64;
            qb[j] = b0 + j * 128 * 64;
          });
        } else {
          static_for<kJ32>([&](auto j) {
            int ra = min(tm * kTile + qrow + 128 * j, m_valid - 1);
            qa[j] = g.A + (int64_t)ra * g.lda + qch * 8;
            int rb = min(tn * kTile + qrow + 128 * j, n_valid - 1);
            if (g.b_rows) rb = g.b_rows[rb];
            qb[j] = g.B + (int64_t)rb * g.ldb + qch * 8;
          });
        }
        // loads K columns 32kt..32kt+31 (row-major: +32kt; tiled: block kt/2,
        // column 32*(kt%2)) into ring stage `buf`
        auto dma32 = [&](int kt, int buf) {
          const int64_t off =
              TILED ? (int64_t)(kt >> 1) * kTileElems + (kt & 1) * 32 : (int64_t)kt * 32;
          char* la = smem + buf * kStage32 + w * 1024;
          static_for<kJ32>([&](auto j) {
            __builtin_amdgcn_global_load_lds((glb_ptr_t)(qa[j] + off),
                                             (lds_ptr_t)(la + j * 8192), 16, 0, 0);
          });
          static_for<kJ32>([&](auto j) {
            __builtin_amdgcn_global_load_lds((glb_ptr_t)(qb[j] + off),
                                             (lds_ptr_t)(la + kTile * 64 + j * 8192), 16, 0,
                                             0);
          });
        };
        const int ra32 = (wm * 128 + fr) * 64;
        const int rb32 = kTile * 64 + (wn * WN + fr) * 64;
        int rc32[2];
        static_for<2>([&](auto t) { rc32[t] = ((2 * t + (lane >> 5)) ^ ((fr >> 2) & 3)) << 4; });
        auto fload32 = [&](int slot, int kt, int t) {
          const char* base = smem + (kt % 5) * kStage32;
          static_for<4>([&](auto i) {
            fa[slot][i] = *(const bf16x8*)(base + ra32 + i * 32 * 64 + rc32[t]);
          });
          static_for<NI>([&](auto i) {
            fb[slot][i] = *(const bf16x8*)(base + rb32 + i * 32 * 64 + rc32[t]);
          });
        };
        // s_waitcnt immediates: vmcnt in bits [3:0], expcnt [6:4] = 7 (no
        // wait), lgkmcnt [11:8] = 0
        constexpr int kPerStep = 2 * kJ32;                        // loads per wave per step
        constexpr int kWaitTwoSteps = 0x0070 | (2 * kPerStep);    // steps kt+2, kt+3 in flight
        constexpr int kWaitThreeSteps = 0x0070 | (3 * kPerStep);
        const int nk = K / 32;
        const int last = nk > 0 ? nk - 1 : 0;  // K = 0 (no valid tokens) still loads stage 0
        dma32(0, 0);
        dma32(min(1, last), 1);
        dma32(min(2, last), 2);
        dma32(min(3, last), 3);
        __builtin_amdgcn_s_waitcnt(kWaitThreeSteps);
        __builtin_amdgcn_s_barrier();
        fload32(0, 0, 0);
        for (int kt = 0; kt < nk; ++kt) {
          fload32(1, kt, 1);
          mfma_sub(0);
          __builtin_amdgcn_sched_group_barrier(kDsRead, kSubReads, 0);
          __builtin_amdgcn_sched_group_barrier(kMfma, kSubMfma, 0);
          __builtin_amdgcn_s_waitcnt(kWaitTwoSteps);
          __builtin_amdgcn_s_barrier();
          // step kt+4 goes to the stage of step kt-1; past the end the last
          // step is loaded again there (never into a stage still in use)
          dma32(min(kt + 4, last), (kt + 4) % 5);
          fload32(0, kt + 1, 0);
          mfma_sub(1);
          __builtin_amdgcn_sched_group_barrier(kDsRead, kSubReads, 1);
          static_for<2 * kJ32>([&](auto) {
            __builtin_amdgcn_sched_group_barrier(kMfma, 1, 1);
            __builtin_amdgcn_sched_group_barrier(kVmem, 1, 1);
          });
        }
        __syncthreads();  // the last (redundant) loads land before LDS is reused
      } else {
      const int nk = K / kBK;

        // ---- Pipeline: while the MFMAs consume LDS buffer kt%2, step kt+1 is
        // landing in the other buffer. The barrier in the middle of step kt
        // (after every wave has read sub-step 3) both publishes step kt+1 and
        // frees buffer kt%2, which immediately receives step kt+2. Sub-step 0
        // of step kt+1 is read right after that barrier, behind the last MFMAs
        // of step kt. __syncthreads() waits for this thread's outstanding LDS
        // loads before the barrier, which is the completion the next step
        // needs. With 8 waves, the two waves of a SIMD interleave their MFMAs
        // with each other's LDS and barrier waits.
        const int last = nk > 0 ? nk - 1 : 0;  // K = 0 (no valid tokens) still loads stage 0
        dma(0, 0);
        __syncthreads();
        dma(min(1, last), 1);
        fload(0, smem, 0);
        for (int kt = 0; kt < nk; ++kt) {
          const char* base = smem + (kt & 1) * kLdsStage;
          fload(1, base, 1);
          mfma_sub(0);
          fload(0, base, 2);
          mfma_sub(1);
          fload(1, base, 3);
          mfma_sub(0);
          __builtin_amdgcn_sched_group_barrier(kDsRead, kSubReads, 0);
          __builtin_amdgcn_sched_group_barrier(kMfma, kSubMfma, 0);
          __builtin_amdgcn_sched_group_barrier(kDsRead, kSubReads, 0);
          __builtin_amdgcn_sched_group_barrier(kMfma, kSubMfma, 0);
          __builtin_amdgcn_sched_group_barrier(kDsRead, kSubReads, 0);
          __builtin_amdgcn_sched_group_barrier(kMfma, kSubMfma, 0);
          __syncthreads();
          dma(min(kt + 2, last), kt & 1);
          fload(0, smem + ((kt + 1) & 1) * kLdsStage, 0);
          mfma_sub(1);
          __builtin_amdgcn_sched_group_barrier(kDsRead, kSubReads, 1);
          static_for<2 * kJ>([&](auto) {
            __builtin_amdgcn_sched_group_barrier(kMfma, 1, 1);
            __builtin_amdgcn_sched_group_barrier(kVmem, 1, 1);
          });
        }
        __syncthreads();  // the last (redundant) loads land before LDS is reused
      }
  } else {
    // ---- K not a multiple of 64: register-staged loads that zero-fill the
    // columns past K. Thread owns rows (tid/8 + 8*kWaves*j), chunk tid%8.
    const int lrow = tid >> 3, lch = tid & 7;
    const uint16_t* pa[kJ];
    const uint16_t* pb[kJ];
#pragma unroll
    for (int j = 0; j < kJ; ++j) {
      int ra = min(tm * kTile + lrow + 8 * kWaves * j, m_valid - 1);
      pa[j] = g.A + (int64_t)ra * g.lda + lch * 8;
      int rb = min(tn * kTile + lrow + 8 * kWaves * j, n_valid - 1);
      if (g.b_rows) rb = g.b_rows[rb];
      pb[j] = g.B + (int64_t)rb * g.ldb + lch * 8;
    }
    const int st_off = lrow * 128 + ((lch ^ swz(lrow)) << 4);  // + 8*kWaves*j rows
    u32x4 ra_[kJ], rb_[kJ];
    auto gload = [&](int kt) {
      const int64_t off = (int64_t)kt * kBK;
#pragma unroll
      for (int j = 0; j < kJ; ++j) {
        if (kt * kBK + lch * 8 >= K) {
          ra_[j] = u32x4{0, 0, 0, 0};
          rb_[j] = u32x4{0, 0, 0, 0};
        } else {
          ra_[j] = *(const u32x4*)(pa[j] + off);
          rb_[j] = *(const u32x4*)(pb[j] + off);
        }
      }
    };
    auto lstore = [&](int buf) {
      char* base = smem + buf * kLdsStage;
#pragma unroll
      for (int j = 0; j < kJ; ++j) {
        *(u32x4*)(base + st_off + j * 8 * kWaves * 128) = ra_[j];
        *(u32x4*)(base + kTile * kBK * 2 + st_off + j * 8 * kWaves * 128) = rb_[j];
      }
    };
    const int nk = (int)ceil_div(K, kBK);
    for (int kt = 0; kt < nk; ++kt) {
      gload(kt);
      lstore(0);
      __syncthreads();
      static_for<4>([&](auto s) {
        fload(0, smem, s);
        mfma_sub(0);
      });
      __syncthreads();
    }
  }

  Frag f{tm, tn, wm, wn, lane, wn * WN};
  epi(acc, f, m_valid, n_valid, smem);
}

#ifndef GRPO_GEMM_WN
#define GRPO_GEMM_WN 64
#endif

template <class Epi, bool TILED>
static void launch_gemm(const GemmArgs& g, const Epi& e, hipStream_t s) {
  int grid = gemm_grid(g.tiles_m, g.tiles_n);
  bool ktail = !TILED && (g.k_dev == nullptr) && (g.K % kBK != 0);
  if (ktail) {
    hipLaunchKernelGGL((k_gemm_bf16<Epi, true, false, 128>), dim3(grid), dim3(256), 0, s, g, e);
  } else {
    constexpr int WN = GRPO_GEMM_WN;
    hipLaunchKernelGGL((k_gemm_bf16<Epi, false, TILED, WN>), dim3(grid),
                       dim3(64 * 2 * (kTile / WN)), 0, s, g, e);
  }
}

void launch_gemm_lse(const GemmArgs& g, const int32_t* y_p, float* zy, float2* ms, int64_t ldms,
                     int64_t V, hipStream_t s) {
  EpiLse e{y_p, zy, ms, ldms, V};
  launch_gemm<EpiLse, false>(g, e, s);
}

void launch_gemm_dz(const GemmArgs& g, const int32_t* y_p, const float* lse_p, const float* g_p,
                    uint16_t* dz, int64_t dz_kt, uint16_t* dzT, int64_t dzT_kt, int64_t V,
                    int64_t v0, hipStream_t s) {
  EpiDz e{y_p, lse_p, g_p, dz, dz_kt, dzT, dzT_kt, V, v0};
  launch_gemm<EpiDz, false>(g, e, s);
}

void launch_gemm_store(const GemmArgs& g, const StoreArgs& a, bool grad_weight, hipStream_t s) {
  EpiStore e{a.acc_buf, a.ld_acc, a.read_acc, a.out, a.ld_out, a.out_bf16, a.add_out,
             a.out_rows, a.m_limit, a.n_limit};
  if (grad_weight)
    launch_gemm<EpiGradWeight, true>(g, EpiGradWeight{e}, s);
  else
    launch_gemm<EpiGradHidden, true>(g, EpiGradHidden{e}, s);
}

}  // namespace grpo
