// Token reorganisation by expert (EaaS §3.3, Fig. 5) and the group-shrink
// compaction of active experts (§4.1): a deterministic stable counting sort of
// the T*k token slots by expert id.
//
//   route_hist     one workgroup per chunk of kRouteChunk slots: LDS histogram
//                  of valid ids -> hist[chunk][e]
//   route_scan     one workgroup: per expert, the exclusive prefix of hist over
//                  chunks (in place), counts, offsets (exclusive scan), and the
//                  compacted ascending list of experts with a non-zero count
//   route_scatter  one workgroup per chunk, each wave owning a contiguous
//                  quarter of it: ranks equal ids inside the wave with ballot
//                  matching, so row = offsets[e] + (earlier chunks) + (earlier
//                  waves) + (earlier steps) + (earlier lanes): stable by slot.
//   route_fused    batches of at most four chunks: the same three steps in one
//                  workgroup (decode sizes, where the launches dominate).
//
// No floating point and no order-dependent atomics: results are bit-exact.
#include "common.h"
#include "internal.h"

namespace eaas {
namespace {

constexpr int kRouteThreads = 256;
constexpr int kScanThreads = 1024;
constexpr int kWavesPerRouteBlock = kRouteThreads / kWave;
constexpr int kSubChunk = kRouteChunk / kWavesPerRouteBlock;

__global__ __launch_bounds__(kRouteThreads) void route_hist_kernel(
    const int32_t* __restrict__ ids, int R, int E, int32_t* __restrict__ hist) {
  __shared__ int cnt[kMaxExperts];
  for (int e = threadIdx.x; e < E; e += kRouteThreads) cnt[e] = 0;
  __syncthreads();
  const int base = blockIdx.x * kRouteChunk;
  const int end = min(base + kRouteChunk, R);
  for (int s = base + threadIdx.x; s < end; s += kRouteThreads) {
    const int id = ids[s];
    if ((unsigned)id < (unsigned)E) atomicAdd(&cnt[id], 1);
  }
  __syncthreads();
  int32_t* h = hist + (size_t)blockIdx.x * E;
  for (int e = threadIdx.x; e < E; e += kRouteThreads) h[e] = cnt[e];
}

// Exclusive scan over a 1024-thread block; returns the prefix, sets *total.
__device__ int block_exclusive_scan_1024(int v, int* s_wave, int* total) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  int incl = v;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int o = __shfl_up(incl, d, kWave);
    if (lane >= d) incl += o;
  }
  if (lane == kWave - 1) s_wave[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    int w = lane < kScanThreads / kWave ? s_wave[lane] : 0;
    int wi = w;
#pragma unroll
    for (int d = 1; d < kScanThreads / kWave; d <<= 1) {
      const int o = __shfl_up(wi, d, kWave);
      if (lane >= d) wi += o;
    }
    if (lane < kScanThreads / kWave) s_wave[lane] = wi - w;
    if (lane == kScanThreads / kWave - 1) s_wave[kScanThreads / kWave] = wi;
  }
  __syncthreads();
  const int res = s_wave[wave] + incl - v;
  *total = s_wave[kScanThreads / kWave];
  __syncthreads();
  return res;
}

__global__ __launch_bounds__(kScanThreads) void route_scan_kernel(
    int32_t* __restrict__ hist, int nblk, int E, int32_t* __restrict__ counts,
    int32_t* __restrict__ offsets, int32_t* __restrict__ active) {
  __shared__ int s_wave[kScanThreads / kWave + 1];
  __shared__ int s_act[kMaxExperts];
  const int e = threadIdx.x;  // E <= 1024 = blockDim
  int c = 0;
  if (e < E) {
    // the loads of a batch of chunks are issued together, ahead of the
    // stores: one memory round trip per kBatch chunks instead of per chunk
    constexpr int kBatch = 16;
    for (int b0 = 0; b0 < nblk; b0 += kBatch) {
      int v[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) v[u] = b0 + u < nblk ? hist[(size_t)(b0 + u) * E + e] : 0;
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        if (b0 + u < nblk) hist[(size_t)(b0 + u) * E + e] = c;  // rows of e in chunks before b
        c += v[u];
      }
    }
  }
  int valid_total;
  const int off = block_exclusive_scan_1024(c, s_wave, &valid_total);
  int n_active;
  const int apos = block_exclusive_scan_1024((e < E && c > 0) ? 1 : 0, s_wave, &n_active);
  if (e < E && c > 0) s_act[apos] = e;
  __syncthreads();
  if (e < E) {
    counts[e] = c;
    offsets[e] = off;
    active[1 + e] = e < n_active ? s_act[e] : 0;
  }
  if (e == 0) {
    offsets[E] = valid_total;
    active[0] = n_active;
  }
}

__global__ __launch_bounds__(kRouteThreads) void route_scatter_kernel(
    const int32_t* __restrict__ ids, int R, int E, int nbits,
    const int32_t* __restrict__ hist, const int32_t* __restrict__ offsets,
    int32_t* __restrict__ perm, int32_t* __restrict__ inv) {
  // next[w][e]: row that the next slot of expert e seen by wave w takes
  __shared__ int next[kWavesPerRouteBlock][kMaxExperts];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int blk = blockIdx.x;
  for (int e = tid; e < E; e += kRouteThreads) {
#pragma unroll
    for (int w = 0; w < kWavesPerRouteBlock; ++w) next[w][e] = 0;
  }
  __syncthreads();
  const int s0 = blk * kRouteChunk + wave * kSubChunk;
  // pass 1: per-wave counts of each expert
  for (int i = 0; i < kSubChunk; i += kWave) {
    const int s = s0 + i + lane;
    const int id = s < R ? ids[s] : -1;
    if ((unsigned)id < (unsigned)E) atomicAdd(&next[wave][id], 1);
  }
  __syncthreads();
  // turn counts into starting rows: offsets[e] + earlier chunks + earlier waves
  for (int e = tid; e < E; e += kRouteThreads) {
    int a = offsets[e] + hist[(size_t)blk * E + e];
#pragma unroll
    for (int w = 0; w < kWavesPerRouteBlock; ++w) {
      const int cw = next[w][e];
      next[w][e] = a;
      a += cw;
    }
  }
  __syncthreads();
  // pass 2: stable ranks, 64 slots per step, steps in slot order
  const uint64_t lt = lanemask_lt();
  for (int i = 0; i < kSubChunk; i += kWave) {
    const int s = s0 + i + lane;
    const int id = s < R ? ids[s] : -1;
    const bool valid = (unsigned)id < (unsigned)E;
    uint64_t peers = ballot(valid);
    for (int b = 0; b < nbits; ++b) {
      const bool bit = (id >> b) & 1;
      const uint64_t m = ballot(bit);
      peers &= bit ? m : ~m;
    }
    int rank = 0;
    if (valid) {
      rank = __popcll(peers & lt);
      const int row = next[wave][id] + rank;
      perm[row] = s;
      inv[s] = row;
    } else if (s < R) {
      inv[s] = -1;
    }
    __builtin_amdgcn_wave_barrier();
    if (valid && rank == 0) next[wave][id] += __popcll(peers);
    __builtin_amdgcn_wave_barrier();
  }
  // rows past the number of valid slots carry no slot
  const int nvalid = offsets[E];
  const int rbeg = max(blk * kRouteChunk, nvalid);
  const int rend = min((blk + 1) * kRouteChunk, R);
  for (int r = rbeg + tid; r < rend; r += kRouteThreads) perm[r] = -1;
}

// Small batches (R <= kFusedMaxSlots = 8192): the three steps in one
// workgroup of 16 waves, with barriers where the separate kernels have
// launch boundaries.  Wave w owns the contiguous slots [w*sub, (w+1)*sub);
// its per-expert counts, turned into starting rows, play the part of the
// per-chunk histogram, so the ranks (and perm, inv) are those of the
// three-kernel path: stable by slot.
constexpr int kFusedWaves = kScanThreads / kWave;
constexpr int kFusedMaxSlots = 4 * kRouteChunk;

__global__ __launch_bounds__(kScanThreads) void route_fused_kernel(
    const int32_t* __restrict__ ids, int R, int E, int nbits, int32_t* __restrict__ counts,
    int32_t* __restrict__ offsets, int32_t* __restrict__ active, int32_t* __restrict__ perm,
    int32_t* __restrict__ inv) {
  __shared__ int next[kFusedWaves * kMaxExperts];  // [w][e], counts then starting rows
  __shared__ int s_wave[kScanThreads / kWave + 1];
  __shared__ int s_act[kMaxExperts];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  for (int i = tid; i < kFusedWaves * E; i += kScanThreads) next[(i / E) * kMaxExperts + i % E] = 0;
  __syncthreads();
  const int sub = (R + kFusedWaves * kWave - 1) / (kFusedWaves * kWave) * kWave;
  const int s0 = wave * sub;
  const int s1 = min(s0 + sub, R);
  int* mine = next + wave * kMaxExperts;
  for (int s = s0 + lane; s < s1; s += kWave) {
    const int id = ids[s];
    if ((unsigned)id < (unsigned)E) atomicAdd(&mine[id], 1);
  }
  __syncthreads();
  // thread e: the expert's count, its offset and the compacted active list
  const int e = tid;  // E <= 1024 = blockDim
  int c = 0;
  if (e < E) {
    for (int w = 0; w < kFusedWaves; ++w) c += next[w * kMaxExperts + e];
  }
  int valid_total;
  const int off = block_exclusive_scan_1024(c, s_wave, &valid_total);
  int n_active;
  const int apos = block_exclusive_scan_1024((e < E && c > 0) ? 1 : 0, s_wave, &n_active);
  if (e < E && c > 0) s_act[apos] = e;
  if (e < E) {
    int a = off;
    for (int w = 0; w < kFusedWaves; ++w) {
      const int cw = next[w * kMaxExperts + e];
      next[w * kMaxExperts + e] = a;
      a += cw;
    }
  }
  __syncthreads();
  if (e < E) {
    counts[e] = c;
    offsets[e] = off;
    active[1 + e] = e < n_active ? s_act[e] : 0;
  }
  if (e == 0) {
    offsets[E] = valid_total;
    active[0] = n_active;
  }
  // stable ranks, 64 slots per step, steps in slot order (as route_scatter)
  const uint64_t lt = lanemask_lt();
  for (int i = s0; i < s0 + sub; i += kWave) {
    const int s = i + lane;
    const int id = s < s1 ? ids[s] : -1;
    const bool valid = (unsigned)id < (unsigned)E;
    uint64_t peers = ballot(valid);
    for (int b = 0; b < nbits; ++b) {
      const bool bit = (id >> b) & 1;
      const uint64_t m = ballot(bit);
      peers &= bit ? m : ~m;
    }
    int rank = 0;
    if (valid) {
      rank = __popcll(peers & lt);
      const int row = mine[id] + rank;
      perm[row] = s;
      inv[s] = row;
    } else if (s < s1) {
      inv[s] = -1;
    }
    __builtin_amdgcn_wave_barrier();
    if (valid && rank == 0) mine[id] += __popcll(peers);
    __builtin_amdgcn_wave_barrier();
  }
  // rows past the number of valid slots carry no slot
  for (int r = valid_total + tid; r < R; r += kScanThreads) perm[r] = -1;
}

}  // namespace

hipError_t launch_route_permute(const int32_t* ids, int R, int E,
                                const eaas_routing& r, int32_t* hist,
                                hipStream_t stream) {
  const int nblk = route_blocks(R);
  int nbits = 1;
  while ((1 << nbits) < E) ++nbits;
  if (R <= kFusedMaxSlots) {
    hipLaunchKernelGGL(route_fused_kernel, dim3(1), dim3(kScanThreads), 0, stream, ids, R, E,
                       nbits, r.counts, r.offsets, r.active, r.perm, r.inv);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(route_hist_kernel, dim3(nblk), dim3(kRouteThreads), 0, stream,
                     ids, R, E, hist);
  hipLaunchKernelGGL(route_scan_kernel, dim3(1), dim3(kScanThreads), 0, stream,
                     hist, nblk, E, r.counts, r.offsets, r.active);
  hipLaunchKernelGGL(route_scatter_kernel, dim3(nblk), dim3(kRouteThreads), 0, stream,
                     ids, R, E, nbits, hist, r.offsets, r.perm, r.inv);
  return hipGetLastError();
}

}  // namespace eaas
