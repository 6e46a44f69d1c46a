// Grouped expert GEMMs over the reorganised token rows (EaaS §3.3 "grouped
// GEMM"; scheduler over the compacted active-expert list of §4.1).
//
// One kernel template serves both projections of the SwiGLU expert:
//   gate/up:  C[r, n] = x[perm[r]/k, :] . W_gate_up[e][n, :]   (rows gathered)
//             epilogue h[r, c] = bf16(silu(C_gate[r, c]) * C_up[r, c])
//   down:     C[r, n] = h[r, :] . W_down[e][n, :]
//             epilogue y[perm[r], n] = w[perm[r]] * C (fp32, rows by slot) or
//                      y[r, n] = C (fp32, rows in permuted order)
//
// Tiles: BM token rows x BN weight rows, BK = 64 along the reduction.  Each of
// the WM x WN waves owns MBW x NBW blocks of 32x32 computed with
// v_mfma_f32_32x32x16_bf16 (src0 = weight rows, src1 = token rows, so a lane
// ends up holding 4 consecutive output columns of one token row).  Operand
// tiles go global -> registers -> LDS (double buffered; the next tile's loads
// are in flight during the current tile's MFMAs).  LDS rows are 128 bytes
// (64 bf16); 16-byte chunk c of row r sits at chunk c ^ (r & 7), so the
// 32-row fragment reads and the row-wise writes are bank-conflict free.
//
// fp8-e4m3 weights (one fp32 scale per 128x128 block) are converted to bf16
// exactly when written to LDS; the MFMA partial sum of every 128-wide K block
// is multiplied by its block scale and added to the fp32 accumulator.
//
// Scheduling: the workgroup reads the compacted active list (group-shrink)
// into LDS once and builds the per-expert M-tile prefix there.  Tile ids are
// ordered expert-major, then weight N-tile, then M-tile, so the M-tiles that
// share one weight tile run back to back; workgroup ids are remapped so each
// XCD (ids congruent mod 8) gets a contiguous range of tiles and its L2 sees
// that reuse.  The grid is sized for the worst case from R and E alone (no
// host readback); surplus workgroups exit after the prologue.
#include "common.h"
#include "internal.h"

namespace eaas {
namespace {

constexpr int kBK = 64;
constexpr int kNumXcd = 8;

enum GemmKind { kGateUp = 0, kDownPlainK = 1, kDownWeightedK = 2 };

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
  const float* w;         // [R] router scores by slot
  int R;                  // slots (T*k)
  int E;                  // resident experts
};

__device__ __forceinline__ float silu_mul(float g, float u) {
  return g / (1.0f + __expf(-g)) * u;
}

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

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;

  // ---- group-shrink: active experts and their M-tile prefix, in LDS once ----
  // routing arrays may come from the caller: clamp every index taken from them
  const int n_active = min(max(p.active[0], 0), p.E);
  {
    // each thread scans PER consecutive entries of the active list (plus the end)
    constexpr int PER = (kMaxExperts + NT) / NT;
    int loc[PER];
    int sum = 0;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int a = tid * PER + i;
      int t = 0;
      if (a < n_active) {
        const int e = min(max(p.active[1 + a], 0), p.E - 1);
        s_exp[a] = e;
        const int beg = min(max(p.offsets[e], 0), p.R);
        const int end = min(max(p.offsets[e + 1], beg), p.R);
        t = ceil_div(end - beg, BM);
      }
      loc[i] = t;
      sum += t;
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
  }
  const int n_tiles_n = p.N / BN;
  const int total = s_tp[n_active] * n_tiles_n;
  const int bid = blockIdx.x;
  if (bid >= total) return;
  int tile = bid;
  {
    const int per = total / kNumXcd;
    if (bid < per * kNumXcd) tile = (bid % kNumXcd) * per + bid / kNumXcd;
  }
  // find active index a with s_tp[a]*n_tiles_n <= tile < s_tp[a+1]*n_tiles_n
  int lo = 0, hi = n_active - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (s_tp[mid] * n_tiles_n <= tile) lo = mid; else hi = mid - 1;
  }
  const int a_idx = lo;
  const int e = s_exp[a_idx];
  const int mt = s_tp[a_idx + 1] - s_tp[a_idx];
  const int local = tile - s_tp[a_idx] * n_tiles_n;
  const int tn = local / mt;
  const int tm = local - tn * mt;
  const int row_beg = min(max(p.offsets[e], 0), p.R);
  const int row_end = min(max(p.offsets[e + 1], row_beg), p.R);
  const int r0 = row_beg + tm * BM;
  const int rows_valid = min(BM, row_end - r0);

  // ---- operand sources ----
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
  // B: weight rows of this tile (gate/up: BN/2 gate rows then the matching up rows)
  const size_t esz = FP8 ? 1 : 2;
  const uint8_t* bexp = p.b + (size_t)e * p.N * p.K * esz;
  constexpr int B_CHUNKS = FP8 ? 4 : 8;  // 16-byte chunks per 64-wide K slice
  const int b_chunk = tid % B_CHUNKS;
  int b_off[B_LOADS];
#pragma unroll
  for (int i = 0; i < B_LOADS; ++i) {
    const int j = tid / B_CHUNKS + i * B_ROWS_PER_PASS;
    int wrow;
    if (GATEUP) wrow = j < BN / 2 ? tn * (BN / 2) + j : p.I + tn * (BN / 2) + (j - BN / 2);
    else wrow = tn * BN + j;
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

  // ---- wave tile ----
  const int wm = wave / WN;
  const int wn = wave % WN;
  const int lrow = lane & 31;
  const int khalf = lane >> 5;
  const int am0 = wm * MBW * 32;  // first token row of this wave inside the tile
  int bn0[NBW];                   // first LDS weight row of each N block
#pragma unroll
  for (int j = 0; j < NBW; ++j) {
    if (GATEUP) {
      constexpr int HB = NBW / 2;
      bn0[j] = j < HB ? wn * HB * 32 + j * 32 : BN / 2 + wn * HB * 32 + (j - HB) * 32;
    } else {
      bn0[j] = wn * NBW * 32 + j * 32;
    }
  }
  // number of 32-row blocks of this wave that hold valid rows (uniform)
  const int mb_live = max(0, min(MBW, ceil_div(rows_valid - am0, 32)));

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
      const float* sexp = p.b_scale + (size_t)e * (p.N / 128) * (p.K / 128);
#pragma unroll
      for (int j = 0; j < NBW; ++j) {
        const int lr = bn0[j];
        int wrow;
        if (GATEUP) wrow = lr < BN / 2 ? tn * (BN / 2) + lr : p.I + tn * (BN / 2) + (lr - BN / 2);
        else wrow = tn * BN + lr;
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

  // ---- epilogue ----
  // acc[i][j][v]: token row am0 + i*32 + lrow, weight row bn0[j] + 8*(v/4) + 4*khalf + v%4
#pragma unroll
  for (int i = 0; i < MBW; ++i) {
    const int rr = am0 + i * 32 + lrow;
    if (i >= mb_live || rr >= rows_valid) continue;
    const int r = r0 + rr;
    if (GATEUP) {
      constexpr int HB = NBW / 2;
      uint16_t* hrow = p.h + (size_t)r * p.I + tn * (BN / 2) + wn * HB * 32;
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
      int orow = r;
      float wt = 1.0f;
      if (KIND == kDownWeightedK) {
        orow = min(max(p.perm[r], 0), p.R - 1);
        wt = p.w[orow];
      }
      float* yrow = p.y + (size_t)orow * p.N + tn * BN + wn * NBW * 32;
#pragma unroll
      for (int j = 0; j < NBW; ++j) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c = j * 32 + 8 * q + 4 * khalf;
          f32x4 v;
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const float a = acc[i][j][4 * q + t];
            v[t] = KIND == kDownWeightedK ? wt * a : a;  // rounded product, stored
          }
          *reinterpret_cast<f32x4*>(yrow + c) = v;
        }
      }
    }
  }
}

template <int KIND, bool FP8, int WM, int WN, int MBW, int NBW>
hipError_t launch_one(const GemmParams& p, int R, int E, hipStream_t stream) {
  constexpr int BM = WM * MBW * 32;
  constexpr int BN = WN * NBW * 32;
  // worst case M-tiles over any routing of R rows onto at most min(E, R) experts
  const long long mt = (long long)(R + BM - 1) / BM + (E < R ? E : R);
  const long long grid = mt * (p.N / BN);
  if (grid <= 0) return hipSuccess;
  if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
  hipLaunchKernelGGL((grouped_gemm_kernel<KIND, FP8, WM, WN, MBW, NBW>), dim3((unsigned)grid),
                     dim3(WM * WN * kWave), 0, stream, p);
  return hipGetLastError();
}

// Tile shapes: prefill-sized batches take 256x256 tiles (4 waves of 128x128);
// decode-sized batches (few rows per expert) take 128-row tiles.
template <int KIND, bool FP8>
hipError_t launch_kind(const GemmParams& p, int R, int E, bool small_m, hipStream_t stream) {
  const bool n256 = (p.N % 256) == 0;
  if (small_m) {
    if (n256) return launch_one<KIND, FP8, 1, 4, 4, 2>(p, R, E, stream);
    return launch_one<KIND, FP8, 1, 2, 4, 2>(p, R, E, stream);
  }
  // fp8 keeps a second (partial-sum) accumulator set, so its tile is half as wide
  if constexpr (!FP8) {
    if (n256) return launch_one<KIND, FP8, 2, 2, 4, 4>(p, R, E, stream);
  }
  return launch_one<KIND, FP8, 2, 2, 4, 2>(p, R, E, stream);
}

}  // namespace

static GemmParams common_params(const FfnArgs& a) {
  GemmParams g{};
  g.perm = a.perm;
  g.k = a.k;
  g.offsets = a.offsets;
  g.active = a.active;
  g.I = a.I;
  g.w = a.topk_weights;
  g.R = a.T * a.k;
  g.E = a.E;
  return g;
}

static bool small_rows(const FfnArgs& a) {
  // decode-sized batches: about one 128-row tile per resident expert or less
  return (long long)a.T * a.k <= 128LL * a.E;
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
  const int R = a.T * a.k;
  const bool sm = small_rows(a);
  if (a.epilogue == kDownWeighted)
    return a.fp8 ? launch_kind<kDownWeightedK, true>(g, R, a.E, sm, stream)
                 : launch_kind<kDownWeightedK, false>(g, R, a.E, sm, stream);
  return a.fp8 ? launch_kind<kDownPlainK, true>(g, R, a.E, sm, stream)
               : launch_kind<kDownPlainK, false>(g, R, a.E, sm, stream);
}

}  // namespace eaas
