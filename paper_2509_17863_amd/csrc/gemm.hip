// Grouped expert GEMMs over the reorganised token rows (EaaS §3.3 "grouped
// GEMM"; scheduler over the compacted active-expert list of §4.1).
//
// Both projections of the SwiGLU expert use the same machinery:
//   gate/up:  C[r, n] = x[perm[r]/k, :] . W_gate_up[e][n, :]   (rows gathered)
//             epilogue h[r, c] = bf16(silu(C_gate[r, c]) * C_up[r, c])
//   down:     C[r, n] = h[r, :] . W_down[e][n, :]
//             epilogue y[perm[r], n] = C (fp32, rows by slot; the combine
//                      applies the router weights) or
//                      y[r, n] = C (fp32, rows in permuted order)
//
// A tile is BM token rows x BN weight rows.  Each of the WM x WN waves owns
// MBW x NBW blocks of 32x32 computed with v_mfma_f32_32x32x16_bf16 (src0 =
// weight rows, src1 = token rows, so a lane ends up holding 4 consecutive
// output columns of one token row).  For gate/up the BN weight rows are BN/2
// gate rows followed by the matching BN/2 up rows, and each wave's blocks pair
// a gate block with the up block of the same columns.
//
// Operands go global -> LDS directly (global_load_lds, 16 B per lane, no VGPR
// staging) through rings of token-row (A) and weight (B) stages; later tiles
// are in flight while one is multiplied.  Waits are explicit vmcnt counts plus
// a bare s_barrier.  Three main loops use this:
//   - bf16 weights: an 8-wave ping-pong in which the two waves of each SIMD
//     alternate between reading a whole K tile's fragments from LDS and
//     issuing its MFMAs (grouped_gemm_pp_kernel);
//   - fp8-e4m3 weights (one fp32 scale per 128x128 block) with bf16
//     activations: the weights stay fp8 in LDS and are converted to bf16
//     (exactly) as fragments are read; each 128-wide K block's MFMA partial
//     sum is scaled and added to the fp32 accumulator
//     (grouped_gemm_dma_kernel);
//   - fp8 weights with fp8 activations (one fp32 scale per row and 128
//     channels): a ping-pong on 16x16x128 block-scaled fp8 MFMAs, each
//     block's partial sum promoted after its K tile (grouped_gemm_w8a8_kernel).
// In the ping-pong loops the multiplying group runs at raised wave priority.
// The fp8-weight down projection runs two 4-wave workgroups per CU.  The
// down epilogues stage each wave's accumulators through LDS so the fp32
// rows go out as whole 256-byte row segments.
// A register-staged loop covers shapes the DMA tiles do not (N not a multiple
// of 256).
// LDS rows are BK elements long; 16-byte chunk c of row r is stored at chunk
// c ^ swz(r) so 32-row fragment reads hit every bank once.
//
// Scheduling: the workgroup reads the compacted active list (group-shrink)
// into LDS once and builds the per-expert M-tile prefix there.  Tile ids are
// ordered expert-major, then in groups of 4 M-tiles, N-tile major and M-tile
// minor inside a group, so tiles that run together share weight and token
// tiles; workgroup ids are remapped so each XCD (ids congruent mod 8) runs 32
// consecutive tiles at a time (its L2 sees that reuse) and the whole GPU one
// window of 256 consecutive tiles (the MALL sees the re-reads across XCDs).
// The grid is sized for the worst case from R and E alone (no host
// readback); surplus workgroups exit after the prologue.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "internal.h"

namespace eaas {
namespace {

#define LDS_AS __attribute__((address_space(3)))
#define CONST_AS __attribute__((address_space(4)))  // read-only global data, scalar loads

constexpr int kNumXcd = 8;
constexpr int kGroupM = 4;  // M-tiles per ordering group inside an expert

enum GemmKind { kGateUp = 0, kDownPlainK = 1, kDownBySlotK = 2 };

struct GemmParams {
  const uint16_t* a;      // gate/up: x [T, lda]; down: h [R, lda]
  const int32_t* perm;    // [R]
  int k;                  // slots per token
  int lda;                // K of this GEMM
  const uint8_t* b;       // weights [E, N, K] (bf16 or fp8 bytes)
  const float* b_scale;   // [E, N/128, K/128] (fp8)
  int N;                  // weight rows per expert
  int K;                  // reduction length
  int I;                  // intermediate size (gate/up: up rows start at I)
  const int32_t* offsets; // [E+1]
  const int32_t* active;  // [E+1]
  uint16_t* h;            // gate/up output [R, I]
  float* y;               // down output [R, N]
  int R;                  // slots (T*k)
  int E;                  // resident experts (groups)
  // server step over several layers: group e is expert e % e_layer of layer
  // e / e_layer, whose weights come from that layer's record instead of b
  const eaas_layer_weights* layers;  // nullptr: one weight array (b, b_scale)
  int e_layer;
  bool down;              // the records' down-projection members
  // fp8 activations: A is fp8 (a8, rows of K bytes) with one fp32 scale per
  // row and 128 channels (a_scale [rows, K/128]); the gate/up epilogue writes
  // h quantized the same way (hq [R, I], hs [R, I/128])
  const uint8_t* a8;
  const float* a_scale;
  uint8_t* hq;
  float* hs;
  // fp8 weights in the tiled layout of tile_weights_fp8 (the ring kernels'
  // weight stages stored contiguously) instead of [E, N, K] row-major
  bool tiled;
};

// Weights of group e ([N, K], bf16 or fp8 bytes of esz each).
__device__ __forceinline__ const uint8_t* group_weights(const GemmParams& p, int e, int esz) {
  if (p.layers == nullptr) return p.b + (size_t)e * p.N * p.K * esz;
  const int L = e / p.e_layer;
  const eaas_layer_weights& lw = p.layers[L];
  return static_cast<const uint8_t*>(p.down ? lw.w_down : lw.w_gate_up) +
         (size_t)(e - L * p.e_layer) * p.N * p.K * esz;
}

// fp8 block scales of group e ([N/128, K/128]).
__device__ __forceinline__ const float* group_scales(const GemmParams& p, int e) {
  const size_t per = (size_t)(p.N / 128) * (p.K / 128);
  if (p.layers == nullptr) return p.b_scale + (size_t)e * per;
  const int L = e / p.e_layer;
  const eaas_layer_weights& lw = p.layers[L];
  return (p.down ? lw.w_down_scale : lw.w_gate_up_scale) + (size_t)(e - L * p.e_layer) * per;
}

struct Tile {
  int e;           // expert
  int tn;          // weight (N) tile
  int r0;          // first permuted row of the tile
  int rows_valid;  // rows of the tile that belong to the expert
};

// silu(g) * u with the hardware exp and reciprocal (a few ulp from the
// correctly rounded value, which moves rare h roundings by one bf16 ulp).
__device__ __forceinline__ float silu_mul(float g, float u) {
  return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u;
}

__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

// One wave-wide 16-byte-per-lane DMA from global memory into LDS: lane l
// reads 16 bytes at base + voff(l) and they land at LDS byte address
// lds + 16*l.  Issued from inline assembly so the compiler adds no waits of
// its own; completion is tracked with explicit vmcnt waits.  `base` and `lds`
// are wave-uniform (SGPRs; `lds` goes to M0).
// The base is passed through readfirstlane so it is held in SGPRs even where
// the compiler cannot prove it uniform (free when it already is).
__device__ __forceinline__ const void* wave_uniform(const void* p) {
  const uint64_t v = reinterpret_cast<uintptr_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<const void*>(((uint64_t)hi << 32) | lo);
}

// NT sets the nontemporal cache policy: used for weight stages that no other
// tile of the launch reads (see stream_weights_once), so they do not displace
// the reused token rows in L2 and the MALL.
template <bool NT = false>
__device__ __forceinline__ void dma16(const void* base, uint32_t voff, uint32_t lds) {
  if constexpr (NT)
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 nt"
                 :: "v"(voff), "s"(wave_uniform(base)), "s"(lds) : "memory");
  else
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :: "v"(voff), "s"(wave_uniform(base)), "s"(lds) : "memory");
}

// Scheduler variant, fixed at build time (the default library is built with
// 0; the other two are built beside it only to reproduce the §4.1 ablation):
//   0  group-shrink: the compacted active-expert list of the routing is read
//      into LDS and the M-tile prefix is scanned over it in parallel;
//   1  the same parallel scan over all E experts, empty ones included;
//   2  the scheduler the paper removes: every workgroup walks the E experts
//      one at a time with one global read of the offsets per expert.
// All three find the same tile for every workgroup id.
#ifndef EAAS_SCHEDULER
#define EAAS_SCHEDULER 0
#endif

// Workgroups are dispatched in id order and round-robin over the XCDs
// (XCD = id mod 8).  The k-th workgroup of XCD x takes tile
//   (k / 32) * 256 + x * 32 + k % 32,
// so the 32 workgroups an XCD runs at once hold 32 consecutive tiles (they
// share token and weight tiles in its L2) and the 256 running on the whole
// GPU hold one window of 256 consecutive tiles, which keeps the weights the
// XCDs re-read within the window in the shared MALL.  Tiles past the last
// whole window keep their ids.
__device__ __forceinline__ int xcd_window_remap(int bid, int total) {
  constexpr int kChunk = 32;
  constexpr int window = kNumXcd * kChunk;
  if (bid >= (total / window) * window) return bid;
  const int x = bid % kNumXcd, kk = bid / kNumXcd;
  return (kk / kChunk) * window + x * kChunk + (kk % kChunk);
}

// Tile `local` of expert e (0 <= local < its M tiles x n_tiles_n).  Inside an
// expert, tiles go in groups of kGroupM M-tiles: N-tile major, M-tile minor
// within a group, so any 32 consecutive tiles (one XCD's workgroups at a
// time) cover <= 4 M-tiles x >= 8 N-tiles and share operands.  (Groups of 4
// rather than 8 halve the token-row re-reads for a quarter more weight
// re-reads; on the prefill shapes that cut the L2 misses by 9-22%.)
template <int BM>
__device__ __forceinline__ void expert_tile(const GemmParams& p, int e, int mt, int local,
                                            int n_tiles_n, Tile& t) {
  const int g = local / (kGroupM * n_tiles_n);
  const int gm = min(kGroupM, mt - g * kGroupM);
  const int lg = local - g * kGroupM * n_tiles_n;
  t.e = e;
  t.tn = lg / gm;
  const int tm = g * kGroupM + (lg - t.tn * gm);
  const int beg = min(max(p.offsets[e], 0), p.R);
  const int end = min(max(p.offsets[e + 1], beg), p.R);
  t.r0 = beg + tm * BM;
  t.rows_valid = min(BM, end - t.r0);
}

#if EAAS_SCHEDULER == 2
// The walking scheduler: one thread walks all E experts twice (the tile
// count, then the expert holding this workgroup's tile), one global read of
// an expert's offsets per step.
template <int BM, int BN, int NT>
__device__ __forceinline__ bool locate_tile(const GemmParams& p, int* s_tp, int* s_exp,
                                            int* s_wave, Tile& t) {
  (void)s_tp; (void)s_exp;
  const int n_tiles_n = p.N / BN;
  auto m_tiles = [&](int e) {
    const int beg = min(max(p.offsets[e], 0), p.R);
    const int end = min(max(p.offsets[e + 1], beg), p.R);
    return ceil_div(end - beg, BM);
  };
  if (threadIdx.x == 0) {
    int all = 0;
    for (int e = 0; e < p.E; ++e) all += m_tiles(e);
    const int total = all * n_tiles_n;
    s_wave[0] = total;
    s_wave[1] = -1;
    if ((int)blockIdx.x < total) {
      const int tile = xcd_window_remap(blockIdx.x, total);
      int before = 0;
      for (int e = 0; e < p.E; ++e) {
        const int mt = m_tiles(e);
        if (tile < (before + mt) * n_tiles_n) {
          s_wave[1] = e;
          s_wave[2] = mt;
          s_wave[3] = tile - before * n_tiles_n;
          break;
        }
        before += mt;
      }
    }
  }
  __syncthreads();
  if (s_wave[1] < 0) return false;
  expert_tile<BM>(p, s_wave[1], s_wave[2], s_wave[3], n_tiles_n, t);
  return true;
}
#else
// Group-shrink schedule: the active list (scheduler 0; every expert for
// scheduler 1) and its M-tile prefix go to LDS once, then this workgroup's
// tile is located by a binary search.  Returns false for surplus groups.
template <int BM, int BN, int NT>
__device__ __forceinline__ bool locate_tile(const GemmParams& p, int* s_tp, int* s_exp,
                                            int* s_wave, Tile& t) {
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  // routing arrays may come from the caller: clamp every index taken from them
  const int n_active = EAAS_SCHEDULER == 1 ? p.E : min(max(p.active[0], 0), p.E);
  constexpr int PER = (kMaxExperts + NT) / NT;  // entries per thread (plus the end)
  int loc[PER];
  int sum = 0;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int a = tid * PER + i;
    int c = 0;
    if (a < n_active) {
      const int e = EAAS_SCHEDULER == 1 ? a : min(max(p.active[1 + a], 0), p.E - 1);
      s_exp[a] = e;
      const int beg = min(max(p.offsets[e], 0), p.R);
      const int end = min(max(p.offsets[e + 1], beg), p.R);
      c = ceil_div(end - beg, BM);
    }
    loc[i] = c;
    sum += c;
  }
  int incl = sum;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int o = __shfl_up(incl, d, kWave);
    if (lane >= d) incl += o;
  }
  if (lane == kWave - 1) s_wave[wave] = incl;
  __syncthreads();
  int before = 0;
#pragma unroll
  for (int w = 0; w < NT / kWave; ++w) before += (w < wave) ? s_wave[w] : 0;
  int run = before + incl - sum;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int a = tid * PER + i;
    if (a <= n_active) s_tp[a] = run;
    run += loc[i];
  }
  __syncthreads();
  const int n_tiles_n = p.N / BN;
  const int total = s_tp[n_active] * n_tiles_n;
  const int bid = blockIdx.x;
  if (bid >= total) return false;
  const int tile = xcd_window_remap(bid, total);
  // the last slot whose prefix is <= tile (empty experts of scheduler 1 share
  // their successor's prefix and are passed over)
  int lo = 0, hi = n_active - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (s_tp[mid] * n_tiles_n <= tile) lo = mid; else hi = mid - 1;
  }
  expert_tile<BM>(p, s_exp[lo], s_tp[lo + 1] - s_tp[lo], tile - s_tp[lo] * n_tiles_n, n_tiles_n,
                  t);
  return true;
}
#endif

// Weight row (of the expert's [N, K] matrix) held by LDS row j of an N tile.
template <bool GATEUP, int BN>
__device__ __forceinline__ int weight_row(const GemmParams& p, int tn, int j) {
  if (GATEUP) return j < BN / 2 ? tn * (BN / 2) + j : p.I + tn * (BN / 2) + (j - BN / 2);
  return tn * BN + j;
}

// First LDS weight row of N block j of wave column wn.
template <bool GATEUP, int BN, int NBW>
__device__ __forceinline__ int block_row(int wn, int j) {
  if (GATEUP) {
    constexpr int HB = NBW / 2;
    return j < HB ? wn * HB * 32 + j * 32 : BN / 2 + wn * HB * 32 + (j - HB) * 32;
  }
  return wn * NBW * 32 + j * 32;
}

// Output row and router weight of each of the lane's token rows, loaded
// before the main loop so the epilogue's stores do not wait on them.
template <int MBW>
struct RowInfo {
  int orow[MBW];
};

template <int KIND, int MBW>
__device__ __forceinline__ RowInfo<MBW> row_info(const GemmParams& p, const Tile& t, int am0,
                                                 int mb_live) {
  RowInfo<MBW> ri;
  const int lrow = threadIdx.x & 31;
#pragma unroll
  for (int i = 0; i < MBW; ++i) {
    const int rr = am0 + i * 32 + lrow;
    const int r = t.r0 + (rr < t.rows_valid ? rr : 0);
    ri.orow[i] = r;
    if (KIND == kDownBySlotK && i < mb_live) ri.orow[i] = min(max(p.perm[r], 0), p.R - 1);
  }
  return ri;
}

// acc[i][j][v]: token row am0 + i*32 + lane%32, weight row
// block_row(j) + 8*(v/4) + 4*(lane/32) + v%4.
template <int KIND, int BN, int MBW, int NBW>
__device__ __forceinline__ void epilogue(const GemmParams& p, const Tile& t, int wn, int am0,
                                         int mb_live, const RowInfo<MBW>& ri,
                                         const f32x16 (&acc)[MBW][NBW]) {
  const int lane = threadIdx.x & (kWave - 1);
  const int lrow = lane & 31;
  const int khalf = lane >> 5;
#pragma unroll
  for (int i = 0; i < MBW; ++i) {
    const int rr = am0 + i * 32 + lrow;
    if (i >= mb_live || rr >= t.rows_valid) continue;
    const int r = t.r0 + rr;
    if (KIND == kGateUp) {
      constexpr int HB = NBW / 2;
      uint16_t* hrow = p.h + (size_t)r * p.I + t.tn * (BN / 2) + wn * HB * 32;
#pragma unroll
      for (int j = 0; j < HB; ++j) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c = j * 32 + 8 * q + 4 * khalf;
          const f32x16 g = acc[i][j];
          const f32x16 u = acc[i][j + HB];
          u32x2 v;
          v[0] = pack_bf16x2(silu_mul(g[4 * q + 0], u[4 * q + 0]), silu_mul(g[4 * q + 1], u[4 * q + 1]));
          v[1] = pack_bf16x2(silu_mul(g[4 * q + 2], u[4 * q + 2]), silu_mul(g[4 * q + 3], u[4 * q + 3]));
          *reinterpret_cast<u32x2*>(hrow + c) = v;
        }
      }
    } else {
      const int orow = ri.orow[i];
      float* yrow = p.y + (size_t)orow * p.N + t.tn * BN + wn * NBW * 32;
#pragma unroll
      for (int j = 0; j < NBW; ++j) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c = j * 32 + 8 * q + 4 * khalf;
          f32x4 v;
#pragma unroll
          for (int u = 0; u < 4; ++u) v[u] = acc[i][j][4 * q + u];
          *reinterpret_cast<f32x4*>(yrow + c) = v;
        }
      }
    }
  }
}

// Down projection epilogue through LDS.  In the MFMA layout a store
// instruction writes 32-byte pieces of 32 different rows (lanes l and l+32
// hold neighbouring 4-column runs of token row l%32), and the fp32 staging
// rows of a down tile are scattered slots: the stores then cost more than
// the tile's last K tiles.  Here each wave passes its accumulators, one
// 32-row block at a time, through a private LDS region and stores whole
// rows of its columns: with NBW = 2 one instruction writes 4 rows x 256
// contiguous bytes.  The values stored are those of `epilogue` (the fp32
// accumulators), bit for bit.  Every wave must have finished
// the main loop's LDS reads (and its DMA must have landed) before any wave
// calls this: the callers reach it after the loop's last barrier.
template <int NBW>
constexpr int kRowsLdsBytes = 32 * (NBW * 32 + 4) * 4;  // one wave's region

template <int KIND, int BN, int MBW, int NBW>
__device__ __forceinline__ void epilogue_rows_lds(const GemmParams& p, const Tile& t, int wn,
                                                  int am0, int mb_live, const RowInfo<MBW>& ri,
                                                  const f32x16 (&acc)[MBW][NBW],
                                                  LDS_AS float* buf) {
  static_assert(KIND != kGateUp, "down projection only");
  constexpr int COLS = NBW * 32;     // the wave's columns
  constexpr int LD = COLS + 4;       // LDS row stride in floats: 16-byte pad against bank conflicts
  constexpr int LPR = COLS / 4;      // lanes per row when reading 16 bytes each
  constexpr int RPI = kWave / LPR;   // rows per read / store instruction
  static_assert(LPR * 4 == COLS && RPI * LPR == kWave && 32 % RPI == 0, "row layout");
  // the lane id from mbcnt, so that threadIdx need not stay live through the loop
  const int lane = __lane_id();
  const int lrow = lane & 31;
  const int khalf = lane >> 5;
  const int rl = lane / LPR;
  const int cl = (lane % LPR) * 4;
  float* ybase = p.y + t.tn * BN + wn * COLS + cl;
#pragma unroll
  for (int i = 0; i < MBW; ++i) {
    if (i >= mb_live) continue;
#pragma unroll
    for (int j = 0; j < NBW; ++j) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        f32x4 v;
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = acc[i][j][4 * q + u];
        *reinterpret_cast<LDS_AS f32x4*>(buf + lrow * LD + j * 32 + 8 * q + 4 * khalf) = v;
      }
    }
    // a wave's LDS operations complete in order: the reads below see the
    // writes above, and the next block's writes follow these reads
#pragma unroll
    for (int s = 0; s < 32 / RPI; ++s) {
      const int m = s * RPI + rl;
      const f32x4 v = *reinterpret_cast<const LDS_AS f32x4*>(buf + m * LD + cl);
      const int orow = __shfl(ri.orow[i], m);  // lane m holds row m's destination
      // non-temporal: the combine reads the staging once, after this launch
      if (am0 + i * 32 + m < t.rows_valid)
        __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(ybase + (size_t)orow * p.N));
    }
  }
}

// ============================================================================
// bf16 weights: LDS-DMA ring
// ============================================================================
// XOR swizzle of the 16-byte chunks of an LDS row.  A fragment read has 8
// lanes (128-byte bank lines) or 16 lanes (256-byte bank lines) in flight per
// cycle, reading one chunk column of consecutive rows; the swizzle puts those
// rows' chunks on distinct banks in both cases.
template <int ROW_BYTES>
__device__ __forceinline__ int swz(int row) {
  static_assert(ROW_BYTES == 64 || ROW_BYTES == 128 || ROW_BYTES == 256, "LDS row size");
  if (ROW_BYTES == 256) return row & 15;                         // 16 chunks
  if (ROW_BYTES == 128) return (row & 7) ^ ((row >> 3) & 1);     // 8 chunks
  return ((row >> 1) & 3) ^ ((row >> 3) & 1);                    // 4 chunks
}

// Global sources of a tile's DMA (shared by the full- and partial-tile loops).
template <int A_INST, int B_INST>
struct DmaSrc {
  const char* a;             // A base (bytes); K tile kt starts kt*BK*2 bytes further
  const char* b;             // B base of the tile (bytes)
  uint32_t b_kstride;        // bytes from one B stage's K position to the next
  uint32_t a_off[A_INST];    // per-lane byte offsets of this lane's DMA rows
  uint32_t b_off[B_INST];
  uint32_t lds;              // LDS byte address of stage 0
  int wave;
};

// 8 fp8-e4m3 values -> 8 bf16 (exact).
__device__ __forceinline__ bf16x8 fp8x8_to_bf16(u32x2 q) {
  bf16x2 v0 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(q[0], 1.0f, false);
  bf16x2 v1 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(q[0], 1.0f, true);
  bf16x2 v2 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(q[1], 1.0f, false);
  bf16x2 v3 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(q[1], 1.0f, true);
  return bf16x8{v0[0], v0[1], v1[0], v1[1], v2[0], v2[1], v3[0], v3[1]};
}

template <int KIND, int BK, int SA, int SB, int BSPAN, int NW, int BM, int BN, int MBW, int NBW,
          bool FULL, bool FP8>
struct DmaLoop {
  static constexpr int RB = BK * 2;            // bytes per LDS row of A (bf16)
  static constexpr int CH = RB / 16;           // 16-byte chunks per A row
  static constexpr int RPI = kWave / CH;       // A rows per wave DMA instruction (1 KiB)
  // A B stage spans BSPAN K tiles, so an fp8 weight row is fetched as whole
  // 128-byte lines (BK = 64, BSPAN = 2) while the token rows stay in BK tiles.
  static constexpr int BTB = FP8 ? BK : 2 * BK;  // bytes of one K tile of a B row
  static constexpr int BRB = BTB * BSPAN;        // bytes per LDS row of a B stage
  static constexpr int BCH = BRB / 16;
  static constexpr int BRPI = kWave / BCH;
  // DMA instruction g (of NA for A, NB for B) covers rows [g*RPI, (g+1)*RPI);
  // wave w issues g = w + NW*q.  When NW does not divide NA, the surplus
  // slots repeat the last instruction (rewriting identical bytes), so every
  // wave issues the same count and the vmcnt arithmetic stays uniform.
  static constexpr int NA = BM / RPI;
  static constexpr int NB = BN / BRPI;
  static_assert(NA * RPI == BM && NB * BRPI == BN, "DMA rows");
  static constexpr int A_INST = (NA + NW - 1) / NW;
  static constexpr int B_INST = (NB + NW - 1) / NW;
  static __device__ __forceinline__ int a_inst(int wave, int q) { return min(wave + NW * q, NA - 1); }
  static __device__ __forceinline__ int b_inst(int wave, int q) { return min(wave + NW * q, NB - 1); }
  static constexpr int INST = A_INST + B_INST;
  // LDS: a ring of SA token-row (A) stages, then a ring of SB weight (B)
  // stages of BSPAN K tiles each.  SB > SA gives the weights, which stream
  // from HBM, more K tiles of flight time than the token rows, which mostly
  // hit L2; BSPAN = 2 (with SA = SB = 2) gives them two.
  static constexpr int A_BYTES = BM * RB;
  static constexpr int B_BYTES = BN * BRB;
  static constexpr int B_BASE = SA * A_BYTES;
  static constexpr int LDS_BYTES = SA * A_BYTES + SB * B_BYTES;
  static constexpr int KK = BK / 16;           // MFMA k-steps per tile
  static constexpr int TILES_PER_SCALE = 128 / BK;  // fp8: K tiles per scale block
  static_assert(KK % 2 == 0, "fragment double buffering alternates sets");
  static_assert(SA >= 2 && SB >= 2 && SA <= 4 && SB <= 4, "ring depths");
  static_assert(BSPAN == 1 || (BSPAN == 2 && FP8 && SA == 2 && SB == 2), "B stage span");
  static_assert(!FP8 || 128 % BK == 0, "fp8 scale blocks hold whole K tiles");

  struct Frags {
    bf16x8 a[MBW];
    bf16x8 b[NBW];
  };

  using Src = DmaSrc<A_INST, B_INST>;

  // DMA instruction q (0..INST-1): the A part loads K tile ka, the B part B
  // stage kb (K tiles kb*BSPAN ..), each into its ring slot; ka >= nk or
  // kb outside [0, nb) issue nothing.
  static __device__ __forceinline__ void issue_one(const Src& s, int ka, int kb, int nk, int nb,
                                                   int q) {
    if (q < A_INST) {
      if (ka < nk)
        dma16(s.a + ka * BK * 2, s.a_off[q],
              s.lds + (ka % SA) * A_BYTES + a_inst(s.wave, q) * RPI * RB);
    } else {
      if (kb >= 0 && kb < nb)
        dma16(s.b + (size_t)kb * s.b_kstride, s.b_off[q - A_INST],
              s.lds + B_BASE + (kb % SB) * B_BYTES + b_inst(s.wave, q - A_INST) * BRPI * BRB);
    }
  }

  static __device__ __forceinline__ void issue_a(const Src& s, int kt, int nk) {
#pragma unroll
    for (int q = 0; q < A_INST; ++q) issue_one(s, kt, -1, nk, 0, q);
  }
  static __device__ __forceinline__ void issue_b(const Src& s, int kb, int nb) {
#pragma unroll
    for (int q = A_INST; q < INST; ++q) issue_one(s, 0, kb, 0, nb, q);
  }

  // B fragment of k-step kk from the B stage at `bsrc`: bf16 rows use the A
  // layout; fp8 rows hold BSPAN K tiles of BK bytes (16-byte chunk kk of K
  // tile part `kp`, 8-byte half per lane half), converted to bf16 here.
  static __device__ __forceinline__ void load_b(const LDS_AS char* bsrc, int kk, int kp, int coff,
                                                const int (&b_lane_off)[NBW], int sb_l,
                                                Frags& f) {
    if constexpr (FP8) {
      const int khalf = (threadIdx.x & 63) >> 5;
      const int boff = (((kp * KK + kk) ^ sb_l) << 4) + khalf * 8;
#pragma unroll
      for (int j = 0; j < NBW; ++j)
        f.b[j] = fp8x8_to_bf16(*reinterpret_cast<const LDS_AS u32x2*>(bsrc + b_lane_off[j] + boff));
    } else {
#pragma unroll
      for (int j = 0; j < NBW; ++j)
        f.b[j] = *reinterpret_cast<const LDS_AS bf16x8*>(bsrc + b_lane_off[j] + coff);
    }
  }

  static __device__ __forceinline__ void load_a(const LDS_AS char* asrc, int coff, int i,
                                                int a_lane_off, int mb_live, Frags& f) {
    if (FULL || i < mb_live)
      f.a[i] = *reinterpret_cast<const LDS_AS bf16x8*>(asrc + a_lane_off + i * 32 * RB + coff);
  }

  // MFMAs of row block i; ZERO starts the accumulation from 0 (the first
  // k-step of an fp8 scale block) instead of reading the accumulator.
  template <bool ZERO = false>
  static __device__ __forceinline__ void mma_row(const Frags& f, int i, int mb_live,
                                                 f32x16 (&acc)[MBW][NBW]) {
    if (FULL || i < mb_live)
#pragma unroll
      for (int j = 0; j < NBW; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.b[j], f.a[i],
                                                            ZERO ? f32x16{} : acc[i][j], 0, 0, 0);
  }

  // Wait until this wave's DMA of K tile kt+1 (both parts) has landed.  Loads
  // complete in issue order for vmcnt, so the wait allows exactly the
  // instructions issued after the later of the two parts.  Issue order:
  // iteration i (tile i's first k-step) issues A(i+SA-1), then B(i+SB-1),
  // each only if it exists; the prologue runs iterations -(max(SA,SB)-1) ..
  // -1 the same way.  after_count(rem) counts, for a tile followed by `rem`
  // more (3 stands for "3 or more": no ring looks further ahead), the
  // instructions issued after the later of A(kt+1), B(kt+1) by the end of
  // iteration kt.  BSPAN == 2: iteration i issues A(i+1), then on even i B
  // stage i/2+1; after A(kt+1) comes that B stage when kt is even (B stage
  // (kt+1)/2, needed when kt is odd, was issued before A(kt)).  kt = -1 is
  // the prologue's wait for tile 0.
  static constexpr int after_count(int rem) {
    const int nk_rel = 1 + rem;                 // K tiles from kt on
    const int j = 2 - (SA < SB ? SA : SB);      // iteration of the later part
    int n = 0;
    if (SA < SB && j + SB - 1 >= 0 && j + SB - 1 < nk_rel) n += B_INST;  // B after A(kt+1)
    for (int i = j + 1; i <= 0; ++i) {
      if (i + SA - 1 >= 0 && i + SA - 1 < nk_rel) n += A_INST;
      if (i + SB - 1 >= 0 && i + SB - 1 < nk_rel) n += B_INST;
    }
    return n;
  }
  static __device__ __forceinline__ void wait_next(int kt, int nk) {
    const int rem = nk - 1 - kt;  // K tiles from kt+1 on
    if constexpr (BSPAN == 2) {
      if (kt >= 0 && (kt & 1) == 0 && kt + 2 < nk) wait_vmcnt<B_INST>();
      else wait_vmcnt<0>();
    } else {
      if (rem >= 3) wait_vmcnt<after_count(3)>();
      else if (rem == 2) wait_vmcnt<after_count(2)>();
      else wait_vmcnt<after_count(1)>();
    }
  }

  // One K tile.  k-step 0: its MFMAs interleaved with the DMA of A tile
  // kt+SA-1 and B tile kt+SB-1 (into the stages tile kt-1 used, released by
  // the previous barrier) and the fragment reads of the next k-step.  Last
  // k-step: half the MFMAs, then the tile boundary (wait for tile kt+1,
  // barrier, first fragments of tile kt+1), then the other half.  The barrier
  // also certifies that every wave finished reading tile kt, so its stages
  // may be refilled during tile kt+1.  FRESH: the tile starts an fp8 scale
  // block, so its first k-step overwrites the partial sums.
  template <bool FRESH>
  static __device__ __forceinline__ void tile(const LDS_AS char* smem, const Src& s, int nk,
                                              int kt, int a_lane_off,
                                              const int (&b_lane_off)[NBW], int s_l, int sb_l,
                                              int mb_live, Frags (&f)[2],
                                              f32x16 (&mac)[MBW][NBW]) {
    const int khalf = (threadIdx.x & 63) >> 5;
    auto coff = [&](int kk) { return (((2 * kk + khalf) ^ s_l) << 4); };
    const LDS_AS char* asrc = smem + (kt % SA) * A_BYTES;
    const LDS_AS char* bsrc = smem + B_BASE + ((kt / BSPAN) % SB) * B_BYTES;
    const int kp = kt % BSPAN;
    const int nb = (nk + BSPAN - 1) / BSPAN;
    const int ka = kt + SA - 1;
    const int kb = kp == 0 ? kt / BSPAN + SB - 1 : -1;  // B stages start on even tiles
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      Frags& fa = f[kk & 1];
      Frags& fb = f[(kk + 1) & 1];
      if (kk + 1 < KK) {
        load_b(bsrc, kk + 1, kp, coff(kk + 1), b_lane_off, sb_l, fb);
#pragma unroll
        for (int i = 0; i < MBW; ++i) {
          load_a(asrc, coff(kk + 1), i, a_lane_off, mb_live, fb);
          if (FRESH && kk == 0) mma_row<true>(fa, i, mb_live, mac);
          else mma_row(fa, i, mb_live, mac);
          if (kk == 0) {
            // spread the INST DMA instructions over the MBW row blocks
#pragma unroll
            for (int q = i * INST / MBW; q < (i + 1) * INST / MBW; ++q)
              issue_one(s, ka, kb, nk, nb, q);
          }
        }
      } else {
#pragma unroll
        for (int i = 0; i < MBW / 2; ++i) mma_row(fa, i, mb_live, mac);
        if (kt + 1 < nk) {
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
          wait_next(kt, nk);
          lds_barrier();
          const LDS_AS char* nasrc = smem + ((kt + 1) % SA) * A_BYTES;
          const LDS_AS char* nbsrc = smem + B_BASE + (((kt + 1) / BSPAN) % SB) * B_BYTES;
          load_b(nbsrc, 0, (kt + 1) % BSPAN, coff(0), b_lane_off, sb_l, fb);
#pragma unroll
          for (int i = 0; i < MBW; ++i) load_a(nasrc, coff(0), i, a_lane_off, mb_live, fb);
        }
#pragma unroll
        for (int i = MBW / 2; i < MBW; ++i) mma_row(fa, i, mb_live, mac);
      }
    }
  }

  // Prologue (in the issue order wait_next assumes), then the K tiles.
  // fp8: the MFMAs of one 128-wide K block (TILES_PER_SCALE tiles) go to
  // `part`, which is then scaled by the block's scale (per N block,
  // sc[j][kb]) and added to `acc`.
  static __device__ __forceinline__ void run(const LDS_AS char* smem, const Src& s, int nk,
                                             int a_lane_off, const int (&b_lane_off)[NBW],
                                             int s_l, int sb_l, int mb_live,
                                             const CONST_AS float* const (&sc)[NBW],
                                             f32x16 (&acc)[MBW][NBW]) {
    const int khalf = (threadIdx.x & 63) >> 5;
    const int coff0 = ((khalf ^ s_l) << 4);
    const int nb = (nk + BSPAN - 1) / BSPAN;
    if constexpr (BSPAN == 2) {
      issue_b(s, 0, nb);
      issue_a(s, 0, nk);
    } else {
      constexpr int S = SA > SB ? SA : SB;
#pragma unroll
      for (int i = -(S - 1); i <= -1; ++i) {
        if (i + SA - 1 >= 0) issue_a(s, i + SA - 1, nk);
        if (i + SB - 1 >= 0) issue_b(s, i + SB - 1, nb);
      }
    }
    wait_next(-1, nk);
    lds_barrier();
    Frags f[2];
    load_b(smem + B_BASE, 0, 0, coff0, b_lane_off, sb_l, f[0]);
#pragma unroll
    for (int i = 0; i < MBW; ++i) load_a(smem, coff0, i, a_lane_off, mb_live, f[0]);

    if constexpr (FP8) {
      f32x16 part[MBW][NBW];
      for (int kt = 0; kt < nk; kt += TILES_PER_SCALE) {
        // the block's scales come through the scalar cache (lgkmcnt), issued
        // before its MFMAs: a vector load here would make the compiler wait
        // for vmcnt(0), draining the DMA ring it does not know about
        const int kb = kt / TILES_PER_SCALE;
        float scale[NBW];
#pragma unroll
        for (int j = 0; j < NBW; ++j) scale[j] = sc[j][kb];
        tile<true>(smem, s, nk, kt, a_lane_off, b_lane_off, s_l, sb_l, mb_live, f, part);
#pragma unroll
        for (int u = 1; u < TILES_PER_SCALE; ++u)
          tile<false>(smem, s, nk, kt + u, a_lane_off, b_lane_off, s_l, sb_l, mb_live, f, part);
#pragma unroll
        for (int j = 0; j < NBW; ++j) {
#pragma unroll
          for (int i = 0; i < MBW; ++i)
            if (FULL || i < mb_live) acc[i][j] += scale[j] * part[i][j];
        }
      }
    } else {
      for (int kt = 0; kt < nk; ++kt)
        tile<false>(smem, s, nk, kt, a_lane_off, b_lane_off, s_l, sb_l, mb_live, f, acc);
    }
  }
};

// OCC: workgroups per CU the launch is sized for (the LDS footprint must
// allow it); it sets the waves per SIMD the registers are budgeted for.
template <int KIND, bool FP8, int BK, int SA, int SB, int BSPAN, int WM, int WN, int MBW, int NBW,
          int OCC>
__global__ __launch_bounds__(WM * WN * kWave)
__attribute__((amdgpu_waves_per_eu(WM * WN * OCC / 4, WM * WN * OCC / 4)))
void grouped_gemm_dma_kernel(GemmParams p) {
  constexpr int NW = WM * WN;
  constexpr int NT = NW * kWave;
  constexpr int BM = WM * MBW * 32, BN = WN * NBW * 32;
  constexpr bool GATEUP = KIND == kGateUp;
  static_assert(!GATEUP || (NBW % 2 == 0), "gate/up pairs gate and up blocks");
  using Full = DmaLoop<KIND, BK, SA, SB, BSPAN, NW, BM, BN, MBW, NBW, true, FP8>;
  using Part = DmaLoop<KIND, BK, SA, SB, BSPAN, NW, BM, BN, MBW, NBW, false, FP8>;
  constexpr int RB = Full::RB, CH = Full::CH, RPI = Full::RPI;
  constexpr int BRB = Full::BRB, BCH = Full::BCH, BRPI = Full::BRPI;

  // the scheduler's tables live in the stage memory until the tile is located
  static_assert(Full::LDS_BYTES >= (2 * kMaxExperts + 1) * 4, "scheduler tables");
  __shared__ __attribute__((aligned(1024))) char smem_raw[Full::LDS_BYTES];
  __shared__ int s_wave[NT / kWave + 1];

  Tile t;
  {
    int* s_tp = reinterpret_cast<int*>(smem_raw);
    int* s_exp = s_tp + kMaxExperts + 1;
    if (!locate_tile<BM, BN, NT>(p, s_tp, s_exp, s_wave, t)) return;
    __syncthreads();  // every lane has its tile before the DMA overwrites the tables
  }

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  // DMA: lane writes 16 bytes at (row lane/CH, physical chunk lane%CH) of its
  // instruction's rows, so it fetches logical chunk (lane%CH) ^ swizzle(row)
  typename Full::Src src;
  src.wave = wave;
  src.a = reinterpret_cast<const char*>(p.a);
  src.b = reinterpret_cast<const char*>(group_weights(p, t.e, FP8 ? 1 : 2));
  // tiled fp8 weights: N tile tn's stages are BN rows x BRB bytes, stored one
  // after the other along K (see tile_weights_fp8)
  const bool tiled = FP8 && BSPAN == 1 && p.tiled;
  src.b_kstride = tiled ? (uint32_t)(BN * BRB) : (uint32_t)BRB;
  if (tiled) src.b += (size_t)t.tn * (p.K / BK) * BN * BRB;
  {
    const int drow = lane / CH;
    const int dpc = lane % CH;
#pragma unroll
    for (int i = 0; i < Full::A_INST; ++i) {
      const int row = Full::a_inst(wave, i) * RPI + drow;
      const int r = t.r0 + (row < t.rows_valid ? row : 0);
      const int src_row = GATEUP ? min(max(p.perm[r], 0), p.R - 1) / p.k : r;
      src.a_off[i] = (uint32_t)(src_row * p.lda + ((dpc ^ swz<RB>(row)) * 8)) * 2u;
    }
  }
  {
    const int drow = lane / BCH;
    const int dpc = lane % BCH;
#pragma unroll
    for (int i = 0; i < Full::B_INST; ++i) {
      const int j = Full::b_inst(wave, i) * BRPI + drow;
      const int chunk = dpc ^ swz<BRB>(j);
      src.b_off[i] = tiled ? (uint32_t)(j * BRB + chunk * 16)
                           : (uint32_t)weight_row<GATEUP, BN>(p, t.tn, j) * (uint32_t)p.K *
                                 (FP8 ? 1u : 2u) + (uint32_t)chunk * 16u;
    }
  }

  const int wm = wave / WN;
  const int wn = wave % WN;
  const int lrow = lane & 31;
  const int am0 = wm * MBW * 32;
  const int a_lane_off = (am0 + lrow) * RB;
  int b_lane_off[NBW];
  const CONST_AS float* sc[NBW];  // per N block: its row of 128x128 scales (wave-uniform)
#pragma unroll
  for (int j = 0; j < NBW; ++j) {
    const int br = block_row<GATEUP, BN, NBW>(wn, j);
    b_lane_off[j] = (br + lrow) * BRB;
    sc[j] = FP8 ? (const CONST_AS float*)wave_uniform(
                      group_scales(p, t.e) +
                      (size_t)(weight_row<GATEUP, BN>(p, t.tn, br) / 128) * (p.K / 128))
                : nullptr;
  }
  const int s_l = swz<RB>(lrow);
  const int sb_l = swz<BRB>(lrow);
  const int mb_live =
      __builtin_amdgcn_readfirstlane(max(0, min(MBW, ceil_div(t.rows_valid - am0, 32))));

  f32x16 acc[MBW][NBW];
#pragma unroll
  for (int i = 0; i < MBW; ++i)
#pragma unroll
    for (int j = 0; j < NBW; ++j) acc[i][j] = f32x16{};

  const RowInfo<MBW> ri = row_info<KIND, MBW>(p, t, am0, mb_live);
  const LDS_AS char* smem = (const LDS_AS char*)smem_raw;  // generic -> LDS address space
  src.lds = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)smem);
  const int nk = p.K / BK;
  if (t.rows_valid == BM)
    Full::run(smem, src, nk, a_lane_off, b_lane_off, s_l, sb_l, mb_live, sc, acc);
  else
    Part::run(smem, src, nk, a_lane_off, b_lane_off, s_l, sb_l, mb_live, sc, acc);

  if constexpr (GATEUP) {
    epilogue<KIND, BN, MBW, NBW>(p, t, wn, am0, mb_live, ri, acc);
  } else {
    // the last K tile ends without a barrier: every wave's fragment reads
    // must be done before the epilogue regions overwrite the stages
    static_assert(NW * kRowsLdsBytes<NBW> <= Full::LDS_BYTES, "epilogue regions");
    __syncthreads();
    epilogue_rows_lds<KIND, BN, MBW, NBW>(
        p, t, wn, am0, mb_live, ri, acc, (LDS_AS float*)(smem_raw + wave * kRowsLdsBytes<NBW>));
  }
}

// ============================================================================
// fp8 weights (and generic shapes): register-staged double buffer, BK = 64
// ============================================================================
constexpr int kBK = 64;

// 16 fp8-e4m3 values -> 16 bf16 (exact), as two 16-byte chunks.
__device__ __forceinline__ void fp8x16_to_bf16(const u32x4 q, u32x4& lo, u32x4& hi) {
  uint32_t o[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    bf16x2 a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(q[i], 1.0f, false);
    bf16x2 b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(q[i], 1.0f, true);
    o[2 * i] = __builtin_bit_cast(uint32_t, a);
    o[2 * i + 1] = __builtin_bit_cast(uint32_t, b);
  }
  lo = u32x4{o[0], o[1], o[2], o[3]};
  hi = u32x4{o[4], o[5], o[6], o[7]};
}

template <int KIND, bool FP8, int WM, int WN, int MBW, int NBW>
__global__ __launch_bounds__(WM * WN * kWave) __attribute__((amdgpu_waves_per_eu(1, 1)))
void grouped_gemm_kernel(GemmParams p) {
  constexpr int NT = WM * WN * kWave;  // threads
  constexpr int BM = WM * MBW * 32;
  constexpr int BN = WN * NBW * 32;
  constexpr bool GATEUP = KIND == kGateUp;
  static_assert(!GATEUP || (NBW % 2 == 0), "gate/up pairs gate and up blocks");
  constexpr int ROWS_PER_PASS = NT / 8;  // rows covered by one 16-byte load per thread
  constexpr int A_LOADS = BM / ROWS_PER_PASS;
  constexpr int B_ROWS_PER_PASS = FP8 ? NT / 4 : NT / 8;
  constexpr int B_LOADS = BN / B_ROWS_PER_PASS;
  static_assert(BM % ROWS_PER_PASS == 0 && BN % B_ROWS_PER_PASS == 0, "tile/thread shape");

  __shared__ bf16x8 As[2][BM * 8];
  __shared__ bf16x8 Bs[2][BN * 8];
  __shared__ int s_tp[kMaxExperts + 1];
  __shared__ int s_exp[kMaxExperts];
  __shared__ int s_wave[NT / kWave + 1];

  Tile t;
  if (!locate_tile<BM, BN, NT>(p, s_tp, s_exp, s_wave, t)) return;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int e = t.e, tn = t.tn, r0 = t.r0, rows_valid = t.rows_valid;

  // A: thread loads chunk (tid % 8) of rows tid/8 + i*ROWS_PER_PASS
  const int a_chunk = tid & 7;
  int a_off[A_LOADS];
#pragma unroll
  for (int i = 0; i < A_LOADS; ++i) {
    const int rr = tid / 8 + i * ROWS_PER_PASS;
    const int r = r0 + (rr < rows_valid ? rr : 0);
    const int src_row = GATEUP ? min(max(p.perm[r], 0), p.R - 1) / p.k : r;
    a_off[i] = src_row * p.lda + a_chunk * 8;
  }
  const size_t esz = FP8 ? 1 : 2;
  const uint8_t* bexp = group_weights(p, e, (int)esz);
  constexpr int B_CHUNKS = FP8 ? 4 : 8;  // 16-byte chunks per 64-wide K slice
  const int b_chunk = tid % B_CHUNKS;
  int b_off[B_LOADS];
#pragma unroll
  for (int i = 0; i < B_LOADS; ++i) {
    const int j = tid / B_CHUNKS + i * B_ROWS_PER_PASS;
    const int wrow = weight_row<GATEUP, BN>(p, tn, j);
    b_off[i] = (wrow * p.K + b_chunk * 16 / (int)esz) * (int)esz;  // bytes
  }

  u32x4 ra[A_LOADS];
  u32x4 rb[B_LOADS];
  auto load_global = [&](int kt) {
    const int k0 = kt * kBK;
#pragma unroll
    for (int i = 0; i < A_LOADS; ++i)
      ra[i] = *reinterpret_cast<const u32x4*>(p.a + a_off[i] + k0);
#pragma unroll
    for (int i = 0; i < B_LOADS; ++i)
      rb[i] = *reinterpret_cast<const u32x4*>(bexp + b_off[i] + (size_t)k0 * esz);
  };
  auto store_lds = [&](int buf) {
#pragma unroll
    for (int i = 0; i < A_LOADS; ++i) {
      const int rr = tid / 8 + i * ROWS_PER_PASS;
      As[buf][rr * 8 + (a_chunk ^ (rr & 7))] = __builtin_bit_cast(bf16x8, ra[i]);
    }
#pragma unroll
    for (int i = 0; i < B_LOADS; ++i) {
      const int j = tid / B_CHUNKS + i * B_ROWS_PER_PASS;
      if (FP8) {
        u32x4 lo, hi;
        fp8x16_to_bf16(rb[i], lo, hi);
        Bs[buf][j * 8 + ((2 * b_chunk) ^ (j & 7))] = __builtin_bit_cast(bf16x8, lo);
        Bs[buf][j * 8 + ((2 * b_chunk + 1) ^ (j & 7))] = __builtin_bit_cast(bf16x8, hi);
      } else {
        Bs[buf][j * 8 + (b_chunk ^ (j & 7))] = __builtin_bit_cast(bf16x8, rb[i]);
      }
    }
  };

  const int wm = wave / WN;
  const int wn = wave % WN;
  const int lrow = lane & 31;
  const int khalf = lane >> 5;
  const int am0 = wm * MBW * 32;  // first token row of this wave inside the tile
  int bn0[NBW];
#pragma unroll
  for (int j = 0; j < NBW; ++j) bn0[j] = block_row<GATEUP, BN, NBW>(wn, j);
  const int mb_live =
      __builtin_amdgcn_readfirstlane(max(0, min(MBW, ceil_div(rows_valid - am0, 32))));

  f32x16 acc[MBW][NBW];
  f32x16 part[FP8 ? MBW : 1][FP8 ? NBW : 1];
#pragma unroll
  for (int i = 0; i < MBW; ++i)
#pragma unroll
    for (int j = 0; j < NBW; ++j) acc[i][j] = f32x16{};
  if (FP8) {
#pragma unroll
    for (int i = 0; i < (FP8 ? MBW : 1); ++i)
#pragma unroll
      for (int j = 0; j < (FP8 ? NBW : 1); ++j) part[i][j] = f32x16{};
  }

  const RowInfo<MBW> ri = row_info<KIND, MBW>(p, t, am0, mb_live);
  const int nk = p.K / kBK;
  load_global(0);
  store_lds(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load_global(kt + 1);
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      const int chunk = 2 * kk + khalf;
      bf16x8 bf[NBW];
#pragma unroll
      for (int j = 0; j < NBW; ++j) {
        const int row = bn0[j] + lrow;
        bf[j] = Bs[cur][row * 8 + (chunk ^ (row & 7))];
      }
#pragma unroll
      for (int i = 0; i < MBW; ++i) {
        if (i < mb_live) {
          const int row = am0 + i * 32 + lrow;
          const bf16x8 af = As[cur][row * 8 + (chunk ^ (row & 7))];
#pragma unroll
          for (int j = 0; j < NBW; ++j) {
            if (FP8)
              part[FP8 ? i : 0][FP8 ? j : 0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                  bf[j], af, part[FP8 ? i : 0][FP8 ? j : 0], 0, 0, 0);
            else
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bf[j], af, acc[i][j], 0, 0, 0);
          }
        }
      }
    }
    if (FP8 && (kt & 1)) {
      // end of a 128-wide K block: acc += scale * partial
      const int kb = kt >> 1;
      const float* sexp = group_scales(p, e);
#pragma unroll
      for (int j = 0; j < NBW; ++j) {
        const int wrow = weight_row<GATEUP, BN>(p, tn, bn0[j]);
        const float sc = sexp[(wrow / 128) * (p.K / 128) + kb];
#pragma unroll
        for (int i = 0; i < MBW; ++i) {
          acc[i][j] += sc * part[FP8 ? i : 0][FP8 ? j : 0];
          part[FP8 ? i : 0][FP8 ? j : 0] = f32x16{};
        }
      }
    }
    if (kt + 1 < nk) store_lds(cur ^ 1);
    __syncthreads();
  }
  epilogue<KIND, BN, MBW, NBW>(p, t, wn, am0, mb_live, ri, acc);
}

// worst case M-tiles over any routing of R rows onto at most min(E, R) experts
inline long long grid_tiles(int R, int E, int BM, int BN, int N) {
  const long long mt = (long long)(R + BM - 1) / BM + (E < R ? E : R);
  return mt * (N / BN);
}

// Whether the bf16 ping-pong and the fp8 x fp8 loop read their weight
// stages with the nontemporal policy: when the R slots fill at most one
// BM-row tile per resident expert on average (a decode-sized batch), each
// weight tile is read once in the launch, and keeping it out of the caches'
// reuse leaves them to the token rows (measured: steps 5% and 8% faster on
// such batches; on the 512-slots-per-expert qwen3 shape, two tiles per
// expert, 1% slower).  Results do not change.
inline bool stream_weights_once(int R, int E, int BM) {
  return (long long)R <= (long long)BM * E;
}

template <int KIND, bool FP8, int WM, int WN, int MBW, int NBW>
hipError_t launch_reg(const GemmParams& p, int R, int E, hipStream_t stream) {
  constexpr int BM = WM * MBW * 32;
  constexpr int BN = WN * NBW * 32;
  const long long grid = grid_tiles(R, E, BM, BN, p.N);
  if (grid <= 0) return hipSuccess;
  if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
  hipLaunchKernelGGL((grouped_gemm_kernel<KIND, FP8, WM, WN, MBW, NBW>), dim3((unsigned)grid),
                     dim3(WM * WN * kWave), 0, stream, p);
  return hipGetLastError();
}

template <int KIND, bool FP8, int BK, int SA, int SB, int BSPAN, int WM, int WN, int MBW, int NBW,
          int OCC = 1>
hipError_t launch_dma(const GemmParams& p, int R, int E, hipStream_t stream) {
  constexpr int BM = WM * MBW * 32, BN = WN * NBW * 32;
  using Loop = DmaLoop<KIND, BK, SA, SB, BSPAN, WM * WN, BM, BN, MBW, NBW, true, FP8>;
  static_assert(OCC * Loop::LDS_BYTES <= 160 * 1024 - OCC * 1024, "workgroups per CU must fit in LDS");
  const long long grid = grid_tiles(R, E, BM, BN, p.N);
  if (grid <= 0) return hipSuccess;
  if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
  // (the fp8 ring reads weights with the default policy: row-major fp8 rows
  // are read 64 bytes of each 128-byte line per K tile, the other half one K
  // tile later, and a nontemporal line may be gone by then (measured:
  // dsv3_decode gate/up 0.21 -> 0.26 ms); on the tiled layout the hint
  // changed nothing, and with Zipf routing it slowed the down projection 7%)
  hipLaunchKernelGGL((grouped_gemm_dma_kernel<KIND, FP8, BK, SA, SB, BSPAN, WM, WN, MBW, NBW, OCC>),
                     dim3((unsigned)grid), dim3(WM * WN * kWave), 0, stream, p);
  return hipGetLastError();
}

// ============================================================================
// bf16 weights, prefill-sized batches: 8-wave ping-pong
// ============================================================================
// 256x256 tiles, BK = 64, 8 waves in two groups of four (one wave of each
// group per SIMD).  Group 0 owns token rows 0-127 of the tile and group 1
// rows 128-255; inside a group wave w4 owns a 64-column slice (two 32-column
// blocks; for gate/up a gate block and the up block of the same columns).
// The groups walk the same K tiles one phase apart.  In an M phase a wave
// issues its share of the operand DMA and reads all four k-steps of its
// fragments of one K tile from LDS into registers; in a C phase it issues
// the 32 MFMAs of those fragments.  While one group multiplies, the other
// reads, so each SIMD's matrix pipe is fed by one of its two waves at a
// time and the LDS reads stay off the MFMA issue path.  Every phase ends
// with an s_barrier of all eight waves:
//   group 0, phase 2t:   M(t): DMA of A tile t+1 (t >= 1), fragments of tile t
//   group 0, phase 2t+1: C(t), then wait until A tile t+1 has landed
//   group 1, phase 2t+1: M(t): DMA of B tile t+2, fragments of tile t, wait
//                        until B tile t+1 has landed
//   group 1, phase 2t+2: C(t)
// A (token rows) has 2 LDS stages and B (weight rows, streamed from HBM) 3.
// A stage is refilled only in the phase after both groups have read it, and
// each tile lands by the barrier before group 0 reads it (A one phase after
// its DMA was issued, B three).  The MFMA order per accumulator is the same
// as in the other GEMM loops: k-steps ascending within a tile, tiles
// ascending, so results do not depend on which loop ran.
template <int KIND, bool NTB>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void grouped_gemm_pp_kernel(GemmParams p) {
  constexpr int BM = 256, BN = 256, BK = 64, MBW = 4, NBW = 2, NT = 512;
  constexpr int RB = BK * 2;   // bytes per LDS row (A and B)
  constexpr int KK = BK / 16;  // MFMA k-steps per K tile
  constexpr int A_BYTES = BM * RB, B_BYTES = BN * RB;
  constexpr int SA = 2, SB = 3;
  constexpr int B_BASE = SA * A_BYTES;
  constexpr int LDS_BYTES = SA * A_BYTES + SB * B_BYTES;  // 160 KiB
  constexpr int INST = 8;      // DMA instructions of one wave per K tile of its operand
  constexpr bool GATEUP = KIND == kGateUp;
  static_assert(INST * 4 * 8 == BM && BM == BN, "4 waves x INST instructions x 8 rows");
  static_assert(LDS_BYTES >= (2 * kMaxExperts + 2 + NT / kWave) * 4, "scheduler tables");
  __shared__ __attribute__((aligned(1024))) char smem_raw[LDS_BYTES];

  Tile t;
  {
    // the scheduler's tables live in the stage memory until the tile is located
    int* s_tp = reinterpret_cast<int*>(smem_raw);
    int* s_exp = s_tp + kMaxExperts + 1;
    int* s_wave = s_exp + kMaxExperts + 1;
    if (!locate_tile<BM, BN, NT>(p, s_tp, s_exp, s_wave, t)) return;
    __syncthreads();  // every lane has its tile before the DMA overwrites the tables
  }

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  const int grp = wave >> 2;  // 0: rows 0-127, streams A; 1: rows 128-255, streams B
  const int w4 = wave & 3;
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)smem_raw);

  // DMA: instruction q of this wave moves rows (w4 + 4q)*8 .. +8 of its
  // group's operand; lane l writes 16 bytes at (row l/8, physical chunk l%8),
  // so it fetches logical chunk (l%8) ^ swizzle(row)
  const char* dbase;
  uint32_t doff[INST];
  {
    const int drow = lane >> 3, dpc = lane & 7;
    if (grp == 0) {
      dbase = reinterpret_cast<const char*>(p.a);
#pragma unroll
      for (int q = 0; q < INST; ++q) {
        const int row = (w4 + 4 * q) * 8 + drow;
        const int r = t.r0 + (row < t.rows_valid ? row : 0);
        const int src_row = GATEUP ? min(max(p.perm[r], 0), p.R - 1) / p.k : r;
        doff[q] = (uint32_t)(src_row * p.lda + ((dpc ^ swz<RB>(row)) * 8)) * 2u;
      }
    } else {
      dbase = reinterpret_cast<const char*>(group_weights(p, t.e, 2));
#pragma unroll
      for (int q = 0; q < INST; ++q) {
        const int j = (w4 + 4 * q) * 8 + drow;
        doff[q] = (uint32_t)weight_row<GATEUP, BN>(p, t.tn, j) * (uint32_t)p.K * 2u +
                  (uint32_t)((dpc ^ swz<RB>(j)) * 16);
      }
    }
  }
  // Ring layouts.  The default: SA token-row stages of BM rows, then SB
  // weight stages.  SMALL (a tile of at most BM/2 rows, which only group 0
  // multiplies): token-row stages of BM/2 rows, and the space freed holds a
  // fourth weight stage, so the weights stream three K tiles ahead.
  struct Ring {
    int a_stage, b_base, sb, a_inst;
  };
  auto ring = [](auto small) {
    constexpr bool SMALL = decltype(small)::value;
    return SMALL ? Ring{A_BYTES / 2, SA * A_BYTES / 2, SB + 1, INST / 2}
                 : Ring{A_BYTES, B_BASE, SB, INST};
  };
  static_assert(SA * A_BYTES / 2 + (SB + 1) * B_BYTES <= LDS_BYTES, "small-tile ring");
  // DMA of K tile kt of this wave's operand into its ring slot
  auto issue = [&](int kt, auto small) {
    constexpr Ring rg = ring(small);
    const char* src = dbase + kt * BK * 2;
    const uint32_t dst = grp == 0 ? lds0 + (kt % SA) * rg.a_stage + w4 * 8 * RB
                                  : lds0 + rg.b_base + (kt % rg.sb) * B_BYTES + w4 * 8 * RB;
    if (grp == 0) {
#pragma unroll
      for (int q = 0; q < rg.a_inst; ++q) dma16(src, doff[q], dst + q * 4 * 8 * RB);
    } else {
#pragma unroll
      for (int q = 0; q < INST; ++q) dma16<NTB>(src, doff[q], dst + q * 4 * 8 * RB);
    }
  };

  const int wn = w4;
  const int lrow = lane & 31;
  const int khalf = lane >> 5;
  const int am0 = grp * MBW * 32;
  const int a_lane_off = (am0 + lrow) * RB;
  int b_lane_off[NBW];
#pragma unroll
  for (int j = 0; j < NBW; ++j) b_lane_off[j] = (block_row<GATEUP, BN, NBW>(wn, j) + lrow) * RB;
  const int s_l = swz<RB>(lrow);  // rows am0 + 32i + lrow share lrow's swizzle
  const int mb_live =
      __builtin_amdgcn_readfirstlane(max(0, min(MBW, ceil_div(t.rows_valid - am0, 32))));

  f32x16 acc[MBW][NBW];
#pragma unroll
  for (int i = 0; i < MBW; ++i)
#pragma unroll
    for (int j = 0; j < NBW; ++j) acc[i][j] = f32x16{};
  const LDS_AS char* smem = (const LDS_AS char*)smem_raw;
  const int nk = p.K / BK;

  auto phase_end = [&]() {
    // keep the scheduler from moving MFMAs or LDS reads across the barrier
    __builtin_amdgcn_sched_barrier(0);
    lds_barrier();
    __builtin_amdgcn_sched_barrier(0);
  };
  // FULL: every row block of the tile holds rows (no per-block checks)
  // SMALL: the small-tile ring (group 1 has no rows to multiply)
  auto main_loop = [&](auto full, auto small) {
    constexpr bool FULL = decltype(full)::value;
    constexpr bool SMALL = decltype(small)::value;
    static_assert(!(FULL && SMALL), "a full tile is not small");
    constexpr Ring rg = ring(small);
    bf16x8 fa[KK][MBW];
    bf16x8 fb[KK][NBW];
    auto load_frags = [&](int kt) {
      const LDS_AS char* asrc = smem + (kt % SA) * rg.a_stage;
      const LDS_AS char* bsrc = smem + rg.b_base + (kt % rg.sb) * B_BYTES;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const int coff = ((2 * kk + khalf) ^ s_l) << 4;
#pragma unroll
        for (int j = 0; j < NBW; ++j)
          fb[kk][j] = *reinterpret_cast<const LDS_AS bf16x8*>(bsrc + b_lane_off[j] + coff);
#pragma unroll
        for (int i = 0; i < MBW; ++i)
          if (FULL || i < mb_live)
            fa[kk][i] =
                *reinterpret_cast<const LDS_AS bf16x8*>(asrc + a_lane_off + i * 32 * RB + coff);
      }
      // the stage may be refilled right after the next barrier
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    };
    // the C phase runs at raised wave priority: its MFMAs win the SIMD's
    // issue arbitration against the other group's fragment reads and DMA
    auto mfmas = [&]() {
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int kk = 0; kk < KK; ++kk)
#pragma unroll
        for (int i = 0; i < MBW; ++i)
          if (FULL || i < mb_live)
#pragma unroll
            for (int j = 0; j < NBW; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[kk][j], fa[kk][i],
                                                                  acc[i][j], 0, 0, 0);
      __builtin_amdgcn_s_setprio(0);
    };

    // prologue: each group's first two K tiles of its operand (SMALL: the
    // weights' first three); tile 0 must have landed before the first barrier
    issue(0, small);
    if (nk > 1) issue(1, small);
    if (SMALL && grp != 0 && nk > 2) {
      issue(2, small);
      wait_vmcnt<2 * INST>();
    } else if (nk > 1) {
      if (grp == 0) wait_vmcnt<rg.a_inst>();
      else wait_vmcnt<INST>();
    } else {
      wait_vmcnt<0>();
    }
    phase_end();
    // both groups pass 2*nk + 1 phase barriers: group 1 idles in the first
    // phase, group 0 in the last
    if (grp == 0) {
      for (int kt = 0; kt < nk; ++kt) {
        if (kt >= 1 && kt + 1 < nk) issue(kt + 1, small);
        load_frags(kt);
        phase_end();
        mfmas();
        wait_vmcnt<0>();  // A tile kt+1 (issued in the previous phase) has landed
        phase_end();
      }
      phase_end();
    } else {
      phase_end();
      for (int kt = 0; kt < nk; ++kt) {
        // B tile kt+3 (SMALL) or kt+2 goes into the stage that tile kt-1
        // used: both groups read it in phases that have ended
        const int ahead = rg.sb - 1;
        if (kt + ahead < nk) issue(kt + ahead, small);
        load_frags(kt);
        // B tile kt+1 has landed; B tiles kt+2 (and kt+3, SMALL) may still be in flight
        if (SMALL && kt + 3 < nk) wait_vmcnt<2 * INST>();
        else if (kt + 2 < nk) wait_vmcnt<INST>();
        else wait_vmcnt<0>();
        phase_end();
        mfmas();
        phase_end();
      }
    }
  };
  // the small-tile ring pays where the weights stream from HBM once
  // (NTB: a decode-sized batch); on gate/up it gained 7-9%, on the down
  // projection and on prefill-sized batches nothing
  if (t.rows_valid == BM) main_loop(std::true_type{}, std::false_type{});
  else if (NTB && GATEUP && t.rows_valid <= BM / 2) main_loop(std::false_type{}, std::true_type{});
  else main_loop(std::false_type{}, std::false_type{});

  // the epilogue's row information is loaded only now: a vector load in
  // the loop would make the compiler wait for vmcnt(0) there
  const RowInfo<MBW> ri = row_info<KIND, MBW>(p, t, am0, mb_live);
  if constexpr (GATEUP) {
    epilogue<KIND, BN, MBW, NBW>(p, t, wn, am0, mb_live, ri, acc);
  } else {
    static_assert(8 * kRowsLdsBytes<NBW> <= LDS_BYTES, "epilogue regions");
    epilogue_rows_lds<KIND, BN, MBW, NBW>(
        p, t, wn, am0, mb_live, ri, acc,
        (LDS_AS float*)(smem_raw + wave * kRowsLdsBytes<NBW>));
  }
}

template <int KIND>
hipError_t launch_pp(const GemmParams& p, int R, int E, hipStream_t stream) {
  const long long grid = grid_tiles(R, E, 256, 256, p.N);
  if (grid <= 0) return hipSuccess;
  if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
  if (stream_weights_once(R, E, 256))
    hipLaunchKernelGGL((grouped_gemm_pp_kernel<KIND, true>), dim3((unsigned)grid), dim3(512), 0,
                       stream, p);
  else
    hipLaunchKernelGGL((grouped_gemm_pp_kernel<KIND, false>), dim3((unsigned)grid), dim3(512), 0,
                       stream, p);
  return hipGetLastError();
}


// ============================================================================
// fp8 weights x fp8 activations
// ============================================================================
// Both operands are e4m3fn with fp32 scales: the weights one per 128x128
// block, the activations one per row and 128 channels.  A K tile is 128
// channels, exactly one scale block of both, and 128 bytes per LDS row as in
// the bf16 loops (same DMA geometry and swizzle).  (The MFMA's internal sums
// are narrower than fp32; promoting every 128 channels keeps their error to
// one K tile's worth.)  As in the bf16 ping-pong kernel, the two groups of
// four waves alternate, phase by phase, between M (fragment reads of a K
// tile, its scales and the group's DMA share) and C (the tile's MFMAs with
// their promotions):
//   group 0, phase 2t:   M(t): DMA of A tile t+1 (t >= 1, with its row
//                        scales), fragments and scales of tile t
//   group 0, phase 2t+1: C(t), then wait until A tile t+1 has landed
//   group 1, phase 2t+1: M(t): DMA of B tile t+2, fragments and scales of
//                        tile t, wait until B tile t+1 has landed
//   group 1, phase 2t+2: C(t)
// A has 2 LDS stages and B 3; a stage is refilled only after both groups have
// read it.  The gate/up epilogue quantizes h per row over the tile's 128 h
// columns (the 4 waves of a group combine their row maxima in LDS).
typedef int i32x8 __attribute__((ext_vector_type(8)));

// One wave-wide 4-byte-per-lane DMA (row scales): lane l's 4 bytes at
// base + voff(l) land at LDS byte address lds + 4*l.
__device__ __forceinline__ void dma4(const void* base, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
               :: "v"(voff), "s"(wave_uniform(base)), "s"(lds) : "memory");
}

// fp8 x fp8 on 16x16x128 block-scaled MFMAs.  One MFMA covers
// a whole 128-channel K tile (one scale block of both operands), so each
// 16x16 block's partial sum lives for a few instructions only and is
// promoted right after its MFMA: acc += (row scale x weight block scale) *
// part.  Without a second accumulator set a wave can hold 96x64 (6 x 4
// blocks of 16x16; token block i, weight block j): it reads 20 KiB of
// fragments per K tile for 24 MFMAs, where a 64x64 wave of 32x32 blocks
// reads 16 KiB for 16.  Lane l supplies row l%16 and K bytes 32*(l/16) .. +32
// of each operand; the result block holds token l%16 and weight columns
// 4*(l/16) .. +3 in lane l.  Tile BM x 256 with BM = 32*MB, 8 waves in two
// groups (token rows 0 .. BM/2-1 and the rest) that alternate M and C
// phases as in the bf16 ping-pong.
// MB = 6 (192-row tiles) for prefill-sized batches, MB = 4 (128 rows) for
// decode-sized ones; the per-block arithmetic is the same, so the two give
// bitwise equal results.
template <int MB>
struct W8Tile {
  static constexpr int BM = 32 * MB, BN = 256, NT = 512, WN = 4, NB = 4;
  static constexpr int RB = 128;
  static constexpr int SA = 2, SB = 3;
  static constexpr int A_BYTES = BM * RB, AS_BYTES = BM * 4, B_BYTES = BN * RB;
  static constexpr int AS_BASE = SA * A_BYTES;
  static constexpr int B_BASE = AS_BASE + SA * AS_BYTES;
  static constexpr int RED_BASE = B_BASE + SB * B_BYTES;
  static constexpr int LDS_BYTES = RED_BASE + BM * WN * 4;
  static constexpr int A_INST = BM / 32;  // 16-byte DMAs of a group-0 wave per K tile (+1 of scales)
  static constexpr int B_INST = 8;        // of a group-1 wave
  static constexpr int AS_CHUNKS = BM / 64;  // 64-row chunks of row scales
};

template <int KIND, int MB, bool NTB>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void grouped_gemm_w8a8_kernel(GemmParams p) {
  using T8 = W8Tile<MB>;
  constexpr int BM = T8::BM, BN = T8::BN, NT = T8::NT, WN = T8::WN, NB = T8::NB, RB = T8::RB;
  constexpr int SA = T8::SA, SB = T8::SB, A_BYTES = T8::A_BYTES, AS_BYTES = T8::AS_BYTES;
  constexpr int B_BYTES = T8::B_BYTES, AS_BASE = T8::AS_BASE, B_BASE = T8::B_BASE;
  constexpr int RED_BASE = T8::RED_BASE, LDS_BYTES = T8::LDS_BYTES;
  constexpr int A_INST = T8::A_INST, B_INST = T8::B_INST;
  constexpr bool GATEUP = KIND == kGateUp;
  static_assert(LDS_BYTES <= 160 * 1024, "LDS");
  static_assert(AS_BASE >= (2 * kMaxExperts + 2 + 2 * (NT / kWave)) * 4, "scheduler tables");
  static_assert(A_INST * 4 * 8 == BM && B_INST * 4 * 8 == BN, "DMA rows");
  __shared__ __attribute__((aligned(1024))) char smem_raw[LDS_BYTES];

  Tile t;
  {
    int* s_tp = reinterpret_cast<int*>(smem_raw);
    int* s_exp = s_tp + kMaxExperts + 1;
    int* s_wave = s_exp + kMaxExperts + 1;
    if (!locate_tile<BM, BN, NT>(p, s_tp, s_exp, s_wave, t)) return;
    __syncthreads();  // every lane has its tile before the DMA overwrites the tables
  }

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  const int grp = wave >> 2;  // 0: rows 0 .. BM/2-1, streams A; 1: the rest, streams B
  const int wn = wave & 3;
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)smem_raw);
  const int nk = p.K / 128;

  auto src_row = [&](int row) {
    const int r = t.r0 + (row < t.rows_valid ? row : 0);
    return GATEUP ? min(max(p.perm[r], 0), p.R - 1) / p.k : r;
  };
  // DMA: instruction q of wave wn moves rows (wn + 4q)*8 .. +8 of the group's
  // operand (lane l: row l/8, physical chunk l%8, logical chunk (l%8) ^
  // swizzle(row)).  Row scales: wave wn writes rows min(wn, chunks-1)*64 .. +64
  // (the last chunk's bytes written twice over, so every wave issues one).
  const char* dbase;
  uint32_t doff[B_INST];
  uint32_t asoff = 0;
  const int as_chunk = min(wn, T8::AS_CHUNKS - 1);
  {
    const int drow = lane >> 3, dpc = lane & 7;
    if (grp == 0) {
      dbase = reinterpret_cast<const char*>(p.a8);
#pragma unroll
      for (int q = 0; q < B_INST; ++q) {
        const int row = (wn + 4 * (q % A_INST)) * 8 + drow;
        doff[q] = (uint32_t)src_row(row) * (uint32_t)p.K + (uint32_t)((dpc ^ swz<RB>(row)) * 16);
      }
      asoff = (uint32_t)src_row(as_chunk * 64 + lane) * (uint32_t)nk * 4u;
    } else {
      dbase = reinterpret_cast<const char*>(group_weights(p, t.e, 1));
#pragma unroll
      for (int q = 0; q < B_INST; ++q) {
        const int j = (wn + 4 * q) * 8 + drow;
        doff[q] = (uint32_t)weight_row<GATEUP, BN>(p, t.tn, j) * (uint32_t)p.K +
                  (uint32_t)((dpc ^ swz<RB>(j)) * 16);
      }
    }
  }
  const char* asbase = reinterpret_cast<const char*>(p.a_scale);
  auto issue = [&](int kt) {
    if (grp == 0) {
      const uint32_t dst = lds0 + (kt % SA) * A_BYTES + wn * 8 * RB;
#pragma unroll
      for (int q = 0; q < A_INST; ++q) dma16(dbase + kt * RB, doff[q], dst + q * 4 * 8 * RB);
      dma4(asbase + kt * 4, asoff, lds0 + AS_BASE + (kt % SA) * AS_BYTES + as_chunk * 256);
    } else {
      const uint32_t dst = lds0 + B_BASE + (kt % SB) * B_BYTES + wn * 8 * RB;
#pragma unroll
      for (int q = 0; q < B_INST; ++q) dma16<NTB>(dbase + kt * RB, doff[q], dst + q * 4 * 8 * RB);
    }
  };

  const int l16 = lane & 15;
  const int kq = lane >> 4;
  const int am0 = grp * (MB * 16);
  const int a_lane_off = (am0 + l16) * RB;
  int b_lane_off[NB];
  const CONST_AS float* sc[NB];  // per weight block: its row of 128x128 scales
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int br = GATEUP ? (j < 2 ? wn * 32 + 16 * j : BN / 2 + wn * 32 + 16 * (j - 2))
                          : wn * 64 + 16 * j;
    b_lane_off[j] = (br + l16) * RB;
    sc[j] = (const CONST_AS float*)wave_uniform(
        group_scales(p, t.e) + (size_t)(weight_row<GATEUP, BN>(p, t.tn, br) / 128) * nk);
  }
  const int s_l = swz<RB>(l16);  // rows am0 + 16i + l16 share l16's swizzle
  const int mb_live =
      __builtin_amdgcn_readfirstlane(max(0, min(MB, ceil_div(t.rows_valid - am0, 16))));
  const LDS_AS char* smem = (const LDS_AS char*)smem_raw;

  // this lane's 32 bytes (chunks 2kq, 2kq+1) of the row at lane_off
  auto frag = [&](const LDS_AS char* base, int lane_off) {
    const int c0 = 2 * kq;
    const u32x4 lo = *reinterpret_cast<const LDS_AS u32x4*>(base + lane_off + ((c0 ^ s_l) << 4));
    const u32x4 hi =
        *reinterpret_cast<const LDS_AS u32x4*>(base + lane_off + (((c0 + 1) ^ s_l) << 4));
    return i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3],
                 (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
  };

  f32x4 acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  auto phase_end = [&]() {
    __builtin_amdgcn_sched_barrier(0);
    lds_barrier();
    __builtin_amdgcn_sched_barrier(0);
  };
  auto main_loop = [&](auto full) {
    constexpr bool FULL = decltype(full)::value;
    i32x8 fa[MB], fb[NB];
    float rsc[MB], wsc[NB];
    // M(kt): the tile's fragments and scales
    auto load_tile = [&](int kt) {
      const LDS_AS char* as = smem + (kt % SA) * A_BYTES;
      const LDS_AS char* bs = smem + B_BASE + (kt % SB) * B_BYTES;
#pragma unroll
      for (int j = 0; j < NB; ++j) fb[j] = frag(bs, b_lane_off[j]);
#pragma unroll
      for (int i = 0; i < MB; ++i)
        if (FULL || i < mb_live) fa[i] = frag(as, a_lane_off + i * 16 * RB);
#pragma unroll
      for (int j = 0; j < NB; ++j) wsc[j] = sc[j][kt];
#pragma unroll
      for (int i = 0; i < MB; ++i)
        if (FULL || i < mb_live)
          rsc[i] = *reinterpret_cast<const LDS_AS float*>(smem + AS_BASE + (kt % SA) * AS_BYTES +
                                                          (am0 + i * 16 + l16) * 4);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    };
    // C(kt): one MFMA per block, each promoted two blocks later (the
    // VALU work runs beside the matrix pipe)
    auto mfmas = [&]() {
      __builtin_amdgcn_s_setprio(1);
      f32x4 pr[3];
      constexpr int NBLK = MB * NB;
#pragma unroll
      for (int b = 0; b < NBLK + 2; ++b) {
        if (b < NBLK) {
          const int i = b / NB, j = b % NB;
          if (FULL || i < mb_live)
            pr[b % 3] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(
                fb[j], fa[i], f32x4{0.0f, 0.0f, 0.0f, 0.0f}, 0, 0, 0, 127, 0, 127);
        }
        if (b >= 2) {
          const int c = b - 2, i = c / NB, j = c % NB;
          if (FULL || i < mb_live) {
            const float f = rsc[i] * wsc[j];
#pragma unroll
            for (int v = 0; v < 4; ++v) acc[i][j][v] += f * pr[c % 3][v];
          }
        }
      }
      __builtin_amdgcn_s_setprio(0);
    };

    constexpr int INST_G0 = A_INST + 1;
    issue(0);
    if (nk > 1) {
      issue(1);
      if (grp == 0) wait_vmcnt<INST_G0>();
      else wait_vmcnt<B_INST>();
    } else {
      wait_vmcnt<0>();
    }
    phase_end();
    if (grp == 0) {
      for (int kt = 0; kt < nk; ++kt) {
        if (kt >= 1 && kt + 1 < nk) issue(kt + 1);
        load_tile(kt);
        phase_end();
        mfmas();
        wait_vmcnt<0>();  // A tile kt+1 (issued in the previous phase) has landed
        phase_end();
      }
      phase_end();
    } else {
      phase_end();
      for (int kt = 0; kt < nk; ++kt) {
        if (kt + 2 < nk) issue(kt + 2);
        load_tile(kt);
        if (kt + 2 < nk) wait_vmcnt<B_INST>();
        else wait_vmcnt<0>();
        phase_end();
        mfmas();
        phase_end();
      }
    }
  };
  if (t.rows_valid == BM) main_loop(std::true_type{});
  else main_loop(std::false_type{});

  // acc[i][j][v]: token row am0 + 16i + l16, weight column 4*kq + v of block j
  if constexpr (GATEUP) {
    // h = bf16(silu(g) * u); per row over the tile's 128 h columns:
    // s = amax / 448, q = e4m3(h / s).  This wave holds 32 of them (gate
    // blocks 0, 1 paired with up blocks 2, 3), 4 per lane per block.
    float* red = reinterpret_cast<float*>(smem_raw + RED_BASE);  // [BM][WN]
    float hv[MB][2][4];
#pragma unroll
    for (int i = 0; i < MB; ++i) {
      float m = 0.0f;
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float h = silu_mul(acc[i][j][v], acc[i][j + 2][v]);
          hv[i][j][v] = __uint_as_float(f32_to_bf16_bits(h) << 16);
          m = fmaxf(m, fabsf(hv[i][j][v]));
        }
      m = fmaxf(m, __shfl_xor(m, 16));
      m = fmaxf(m, __shfl_xor(m, 32));
      if (kq == 0) red[(am0 + i * 16 + l16) * WN + wn] = m;
    }
    __syncthreads();
    const int nkh = p.I / 128;
#pragma unroll
    for (int i = 0; i < MB; ++i) {
      const int rr = am0 + i * 16 + l16;
      if (rr >= t.rows_valid) continue;
      const int r = t.r0 + rr;
      float m = 0.0f;
#pragma unroll
      for (int w = 0; w < WN; ++w) m = fmaxf(m, red[rr * WN + w]);
      const float s = m > 0.0f ? m / 448.0f : 1.0f;
      uint8_t* qrow = p.hq + (size_t)r * p.I + t.tn * (BN / 2) + wn * 32;
#pragma unroll
      for (int j = 0; j < 2; ++j)
        *reinterpret_cast<uint32_t*>(qrow + 16 * j + 4 * kq) =
            pack_e4m3x4(hv[i][j][0] / s, hv[i][j][1] / s, hv[i][j][2] / s, hv[i][j][3] / s);
      if (wn == 0 && kq == 0) p.hs[(size_t)r * nkh + t.tn] = s;
    }
  } else {
    // after the loop's last barrier no wave reads the stages: each wave
    // stages 32 rows (two token blocks) at a time in its own LDS region and
    // stores whole 256-byte row segments
    int orow[MB];
#pragma unroll
    for (int i = 0; i < MB; ++i) {
      const int rr = am0 + i * 16 + l16;
      const int r = t.r0 + (rr < t.rows_valid ? rr : 0);
      orow[i] = r;
      if (KIND == kDownBySlotK && i < mb_live) orow[i] = min(max(p.perm[r], 0), p.R - 1);
    }
    constexpr int COLS = NB * 16, LD = COLS + 4, LPR = COLS / 4, RPI = kWave / LPR;
    static_assert(8 * 32 * LD * 4 <= LDS_BYTES, "epilogue regions");
    static_assert(MB % 2 == 0, "the passes below take token blocks in pairs");
    LDS_AS float* buf = (LDS_AS float*)(smem_raw + wave * (32 * LD * 4));
    const int rl = lane / LPR, cl = (lane % LPR) * 4;
    float* ybase = p.y + t.tn * BN + wn * COLS + cl;
#pragma unroll
    for (int pb = 0; pb < MB / 2; ++pb) {
      if (2 * pb >= mb_live) break;
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        const int i = 2 * pb + h2;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          f32x4 v;
#pragma unroll
          for (int u = 0; u < 4; ++u)
            v[u] = acc[i][j][u];
          *reinterpret_cast<LDS_AS f32x4*>(buf + (16 * h2 + l16) * LD + 16 * j + 4 * kq) = v;
        }
      }
#pragma unroll
      for (int sidx = 0; sidx < 32 / RPI; ++sidx) {
        const int m = sidx * RPI + rl;
        const f32x4 v = *reinterpret_cast<const LDS_AS f32x4*>(buf + m * LD + cl);
        const int o0 = __shfl(orow[2 * pb], m & 15);
        const int o1 = __shfl(orow[2 * pb + 1], m & 15);
        const int o = m < 16 ? o0 : o1;
        if (am0 + pb * 32 + m < t.rows_valid)
          __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(ybase + (size_t)o * p.N));
      }
    }
  }
}

template <int KIND, int MB>
hipError_t launch_w8a8_mb(const GemmParams& p, int R, int E, hipStream_t stream) {
  using T8 = W8Tile<MB>;
  const long long grid = grid_tiles(R, E, T8::BM, T8::BN, p.N);
  if (grid <= 0) return hipSuccess;
  if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
  if (stream_weights_once(R, E, T8::BM))
    hipLaunchKernelGGL((grouped_gemm_w8a8_kernel<KIND, MB, true>), dim3((unsigned)grid),
                       dim3(T8::NT), 0, stream, p);
  else
    hipLaunchKernelGGL((grouped_gemm_w8a8_kernel<KIND, MB, false>), dim3((unsigned)grid),
                       dim3(T8::NT), 0, stream, p);
  return hipGetLastError();
}

// 192-row tiles for prefill-sized batches; 128-row tiles when an expert gets
// about one 128-row tile or less (decode), where taller tiles would only
// stream more empty token rows.  Both give the same bits.
template <int KIND>
hipError_t launch_w8a8(const GemmParams& p, int R, int E, bool small_m, hipStream_t stream) {
  return small_m ? launch_w8a8_mb<KIND, 4>(p, R, E, stream)
                 : launch_w8a8_mb<KIND, 6>(p, R, E, stream);
}

// N-tile width of the fp8-weight ring kernels (launch_kind below): 512 for
// a gate/up matrix whose 2I rows are a multiple of 512, else 256.
inline int fp8_tile_width(bool gateup, int N) { return gateup && N % 512 == 0 ? 512 : 256; }

// Tiled fp8 weights: for expert e, N tile tn (BN rows) and K tile kt (64
// bytes), the BN row slices the ring kernel loads into one weight stage are
// stored contiguously, in the stage's row order (gate/up: the tile's BN/2
// gate rows, then the matching up rows):
//   tiled[((e * N/BN + tn) * K/64 + kt) * BN * 64 + j * 64 + b]
//     = w[e][row(tn, j)][kt * 64 + b]
// One thread per 16-byte chunk of the output.
__global__ __launch_bounds__(256) void tile_weights_fp8_kernel(const uint8_t* __restrict__ w,
                                                               uint8_t* __restrict__ out, int E,
                                                               int N, int K, int I, int BN) {
  const long long chunks = (long long)E * N * K / 16;
  for (long long c = (long long)blockIdx.x * blockDim.x + threadIdx.x; c < chunks;
       c += (long long)gridDim.x * blockDim.x) {
    const long long byte = c * 16;
    const int b = (int)(byte % 64);
    const long long slice = byte / 64;          // (e, tn, kt, j)
    const int j = (int)(slice % BN);
    const long long tk = slice / BN;             // (e, tn, kt)
    const int nkt = K / 64;
    const int kt = (int)(tk % nkt);
    const long long et = tk / nkt;               // (e, tn)
    const int ntn = N / BN;
    const int tn = (int)(et % ntn);
    const int e = (int)(et / ntn);
    const int row = I > 0 ? (j < BN / 2 ? tn * (BN / 2) + j : I + tn * (BN / 2) + (j - BN / 2))
                          : tn * BN + j;
    const u32x4 v = *reinterpret_cast<const u32x4*>(w + ((long long)e * N + row) * K + kt * 64 + b);
    *reinterpret_cast<u32x4*>(out + byte) = v;
  }
}

// Tile shapes (N a multiple of 256 takes the LDS-DMA kernels):
//   bf16: 256x256 tiles, 8 waves of 128x64 in ping-pong, BK=64;
//   fp8 weights, gate/up: 96x512 tiles (a decode batch's ~50-90 rows per
//     expert fit one tile, so the weights stream once), 8 waves of 96x64 --
//     two per SIMD, so one wave's partial-sum scaling (VALU) overlaps the
//     other's MFMAs -- BK=64, 2 token-row stages and 4 weight stages
//     (152 KiB), so 96 KiB of weights per CU are in flight while a tile is
//     multiplied (96x256 with 4 waves and 3+3 stages when N is not a
//     multiple of 512);
//   fp8 weights, down: 96x256 tiles of 4 waves, two workgroups per CU;
//   fp8 weights and activations: 192x256 (prefill) or 128x256 (decode);
//   N not a multiple of 256: register-staged 128-row tiles.
template <int KIND, bool FP8>
hipError_t launch_kind(const GemmParams& p, int R, int E, bool small_m, hipStream_t stream) {
  const bool n256 = (p.N % 256) == 0;
  if constexpr (FP8) {
    // the down projection runs two 4-wave workgroups of 96x256 per CU: twice
    // the tiles of the 512-wide layout (a shorter tail), and two independent
    // barrier domains per CU
    if constexpr (KIND != kGateUp) {
      if (n256) return launch_dma<KIND, true, 64, 2, 3, 1, 1, 4, 3, 2, 2>(p, R, E, stream);
    } else {
      if (p.N % 512 == 0) return launch_dma<KIND, true, 64, 2, 4, 1, 1, 8, 3, 2>(p, R, E, stream);
      if (n256) return launch_dma<KIND, true, 64, 3, 3, 1, 1, 4, 3, 2>(p, R, E, stream);
    }
    if (small_m) return launch_reg<KIND, true, 1, 2, 4, 2>(p, R, E, stream);
    return launch_reg<KIND, true, 2, 2, 4, 2>(p, R, E, stream);
  } else {
    // the ping-pong kernel also beats the register-staged loop on
    // decode-sized batches (its weight stream keeps more bytes in flight)
    if (n256) return launch_pp<KIND>(p, R, E, stream);
    if (small_m) return launch_reg<KIND, false, 1, 2, 4, 2>(p, R, E, stream);
    return launch_reg<KIND, false, 2, 2, 4, 2>(p, R, E, stream);
  }
}

GemmParams common_params(const FfnArgs& a) {
  GemmParams g{};
  g.perm = a.perm;
  g.k = a.k;
  g.offsets = a.offsets;
  g.active = a.active;
  g.I = a.I;
  g.R = a.T * a.k;
  g.E = a.E;
  g.layers = a.layers;
  g.e_layer = a.e_layer;
  g.tiled = a.tiled;
  return g;
}

bool small_rows(const FfnArgs& a) {
  // decode-sized batches: about one 128-row tile per resident expert or less
  return (long long)a.T * a.k <= 128LL * a.E;
}

}  // namespace

hipError_t launch_tile_weights_fp8(const uint8_t* w, uint8_t* out, int E, int N, int K, int I,
                                   hipStream_t stream) {
  const int BN = fp8_tile_width(I > 0, N);
  if (E <= 0 || N % BN || K % 128) return hipErrorInvalidValue;
  const long long chunks = (long long)E * N * K / 16;
  const long long blocks = std::min<long long>((chunks + 255) / 256, 65536);
  hipLaunchKernelGGL(tile_weights_fp8_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, w, out,
                     E, N, K, I, BN);
  return hipGetLastError();
}

hipError_t launch_gate_up(const FfnArgs& a, hipStream_t stream) {
  // [R,H] x [2I,H]^T -> h [R,I]
  GemmParams g = common_params(a);
  g.a = a.x;
  g.lda = a.H;
  g.b = static_cast<const uint8_t*>(a.w_gate_up);
  g.b_scale = a.s_gate_up;
  g.N = 2 * a.I;
  g.K = a.H;
  g.h = a.h;
  const int R = a.T * a.k;
  if (a.act8) {
    g.a8 = a.xq;
    g.a_scale = a.xs;
    g.hq = a.hq;
    g.hs = a.hs;
    return launch_w8a8<kGateUp>(g, R, a.E, small_rows(a), stream);
  }
  return a.fp8 ? launch_kind<kGateUp, true>(g, R, a.E, small_rows(a), stream)
               : launch_kind<kGateUp, false>(g, R, a.E, small_rows(a), stream);
}

hipError_t launch_down(const FfnArgs& a, hipStream_t stream) {
  // [R,I] x [H,I]^T -> y [R,H]
  GemmParams g = common_params(a);
  g.a = a.h;
  g.lda = a.I;
  g.b = static_cast<const uint8_t*>(a.w_down);
  g.b_scale = a.s_down;
  g.N = a.H;
  g.K = a.I;
  g.y = a.y;
  g.down = true;
  const int R = a.T * a.k;
  if (a.act8) {
    g.a8 = a.hq;
    g.a_scale = a.hs;
    return a.epilogue == kDownBySlot ? launch_w8a8<kDownBySlotK>(g, R, a.E, small_rows(a), stream)
                                     : launch_w8a8<kDownPlainK>(g, R, a.E, small_rows(a), stream);
  }
  const bool sm = small_rows(a);
  if (a.epilogue == kDownBySlot)
    return a.fp8 ? launch_kind<kDownBySlotK, true>(g, R, a.E, sm, stream)
                 : launch_kind<kDownBySlotK, false>(g, R, a.E, sm, stream);
  return a.fp8 ? launch_kind<kDownPlainK, true>(g, R, a.E, sm, stream)
               : launch_kind<kDownPlainK, false>(g, R, a.E, sm, stream);
}

}  // namespace eaas
