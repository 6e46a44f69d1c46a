// Dynamic batch of several clients' requests (EaaS §3.3: the server
// aggregates the ready requests of all its clients into one batch, computes,
// and writes each client's weighted sums back into that client's payload).
//
// Both kernels walk the batch with Algorithm 1 of §4 ("Iterate tokens with
// various length of batches"): a static grid whose size does not depend on
// the token counts; the counts are read on the device into shared memory;
// block b starts at token b of the first request, strides by the grid size
// inside a request, and carries the overshoot into the next request, so empty
// requests cost nothing and the load is spread over all blocks without any
// host-side sizing.  Global token g (tokens of earlier requests + index in
// its request) is therefore handled by block g mod gridDim.x.
//
//   seg_gather:  token g of the batch -> row g of the contiguous batch
//                (hidden state, expert ids, router scores); slots of the
//                unused capacity get id -1, so the routing skips them
//   seg_combine: out_b[t] = sum over ascending j of w[s] times the staged row
//                of slot s = g*k+j, in fp32 from +0 without fused multiply-add:
//                bitwise what the single-batch combine writes for token g
#include "common.h"
#include "internal.h"

namespace eaas {
namespace {

constexpr int kSegThreads = 256;

// Count of request b after clamping to the capacity left (the running total
// never exceeds cap, so tokens past the capacity are never touched).
__device__ __forceinline__ int clamp_count(int n, int base, int cap) {
  return max(0, min(n, cap - base));
}

__device__ __forceinline__ void load_counts(const int32_t* num_tokens, int n_seg, int* s_n) {
  for (int b = threadIdx.x; b < n_seg; b += blockDim.x) s_n[b] = max(num_tokens[b], 0);
  __syncthreads();
}

// id_off (optional, per request): valid ids e in [0, e_local) become group
// id_off[b] + e; a negative id_off masks every slot of the request.
__global__ __launch_bounds__(kSegThreads) void seg_gather_kernel(
    const eaas_segment* __restrict__ segs, const int32_t* __restrict__ num_tokens, int n_seg,
    int cap, int H, int k, const int32_t* __restrict__ id_off, int e_local,
    uint16_t* __restrict__ x_cat, int32_t* __restrict__ ids_cat, float* __restrict__ w_cat) {
  __shared__ int s_n[kMaxSegments];
  load_counts(num_tokens, n_seg, s_n);
  const int row_chunks = H / 8;  // 16-byte chunks of a bf16 row
  int token_id = blockIdx.x;
  int base = 0;  // tokens of the requests before b
  for (int b = 0; b < n_seg; ++b) {
    const int n = clamp_count(s_n[b], base, cap);
    if (token_id < n) {
      const eaas_segment sg = segs[b];
      const int off = id_off ? id_off[b] : 0;
      const u32x4* src = static_cast<const u32x4*>(sg.x);
      while (token_id < n) {
        const size_t g = (size_t)base + token_id;
        const u32x4* srow = src + (size_t)token_id * row_chunks;
        u32x4* drow = reinterpret_cast<u32x4*>(x_cat + g * H);
        for (int c = threadIdx.x; c < row_chunks; c += blockDim.x) drow[c] = srow[c];
        for (int j = threadIdx.x; j < k; j += blockDim.x) {
          int id = sg.topk_ids[(size_t)token_id * k + j];
          if (id_off) id = (off >= 0 && (unsigned)id < (unsigned)e_local) ? off + id : -1;
          ids_cat[g * k + j] = id;
          w_cat[g * k + j] = sg.topk_weights[(size_t)token_id * k + j];
        }
        token_id += gridDim.x;
      }
    }
    token_id -= n;
    base += n;
  }
  // unused capacity: slots no expert owns, skipped by the routing
  const size_t first = (size_t)base * k, end = (size_t)cap * k;
  for (size_t i = first + (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < end;
       i += (size_t)gridDim.x * blockDim.x)
    ids_cat[i] = -1;
}

template <bool OUT_FP32>
__global__ __launch_bounds__(kSegThreads) void seg_combine_kernel(
    const eaas_segment* __restrict__ segs, const int32_t* __restrict__ num_tokens, int n_seg,
    int cap, int H, int k, const float* __restrict__ stage, const int32_t* __restrict__ inv,
    const float* __restrict__ w) {
  // products and sums are rounded separately: no fused multiply-add here
#pragma clang fp contract(off)
  __shared__ int s_n[kMaxSegments];
  load_counts(num_tokens, n_seg, s_n);
  int token_id = blockIdx.x;
  int base = 0;
  for (int b = 0; b < n_seg; ++b) {
    const int n = clamp_count(s_n[b], base, cap);
    if (token_id < n) {
      void* out = segs[b].out;
      while (token_id < n) {
        const size_t g = (size_t)base + token_id;
        for (int c = threadIdx.x * 4; c < H; c += blockDim.x * 4) {
          f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
          for (int j = 0; j < k; ++j) {
            const size_t s = g * k + j;
            if (inv[s] < 0) continue;
            const f32x4 v = __builtin_nontemporal_load(
                reinterpret_cast<const f32x4*>(stage + s * H + c));
            const float ws = w[s];
#pragma unroll
            for (int q = 0; q < 4; ++q) acc[q] = acc[q] + ws * v[q];
          }
          if (OUT_FP32) {
            *reinterpret_cast<f32x4*>(static_cast<float*>(out) + (size_t)token_id * H + c) = acc;
          } else {
            u32x2 o;
            o[0] = pack_bf16x2(acc[0], acc[1]);
            o[1] = pack_bf16x2(acc[2], acc[3]);
            *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(out) + (size_t)token_id * H + c) = o;
          }
        }
        token_id += gridDim.x;
      }
    }
    token_id -= n;
    base += n;
  }
}

// Server step, first kernel (one workgroup, thread b = slot b): snapshot the
// flags with system-scope acquire loads, take the ready slots in slot order
// while the running token total fits the capacity (an inclusive scan of the
// ready slots' clamped batch sizes: once it passes the capacity it stays
// past it, so every later ready slot waits for a later step), and lay out the
// taken requests as a dynamic batch: request records, token counts, and the
// group offset of the request's layer.
__global__ __launch_bounds__(kMaxSegments) void slot_snapshot_kernel(
    const eaas_slot* __restrict__ slots, int n_slots, int cap, int n_layers, int e_layer,
    eaas_segment* __restrict__ segs, int32_t* __restrict__ num_tokens,
    int32_t* __restrict__ id_off, int32_t* __restrict__ taken) {
  __shared__ long long s_wave[kMaxSegments / kWave];
  const int b = threadIdx.x;
  const int lane = b & (kWave - 1), wave = b / kWave;
  bool ready = false;
  long long cnt = 0;  // counts are summed in 64 bits: 1024 of them can pass 2^31
  int layer = -1;
  eaas_slot sl{};
  if (b < n_slots) {
    sl = slots[b];
    const int f = __hip_atomic_load(sl.flag, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_SYSTEM);
    if (f == EAAS_SLOT_READY) {
      ready = true;
      layer = sl.header[0];
      cnt = max(0LL, min((long long)sl.header[1], (long long)sl.capacity));
    }
  }
  long long incl = cnt;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const long long o = __shfl_up(incl, d, kWave);
    if (lane >= d) incl += o;
  }
  if (lane == kWave - 1) s_wave[wave] = incl;
  __syncthreads();
  long long run = incl;
  for (int w = 0; w < wave; ++w) run += s_wave[w];
  if (b < n_slots) {
    const bool take = ready && run <= cap;
    taken[b] = take;
    num_tokens[b] = take ? (int)cnt : 0;
    id_off[b] = (layer >= 0 && layer < n_layers) ? layer * e_layer : -1;
    eaas_segment sg;
    sg.x = sl.x;
    sg.topk_ids = sl.topk_ids;
    sg.topk_weights = sl.topk_weights;
    sg.out = sl.x;
    segs[b] = sg;
  }
}

// Server step, last kernel: the taken slots' flags become "server
// computation done", after a system-scope fence over the results (this
// kernel runs after the combine on the same stream).
__global__ __launch_bounds__(kMaxSegments) void slot_complete_kernel(
    const eaas_slot* __restrict__ slots, int n_slots, const int32_t* __restrict__ taken) {
  const int b = threadIdx.x;
  if (b >= n_slots || !taken[b]) return;
  __threadfence_system();
  __hip_atomic_store(slots[b].flag, (int)EAAS_SLOT_DONE, __ATOMIC_RELEASE,
                     __HIP_MEMORY_SCOPE_SYSTEM);
}

// Static grids: sized from the capacity alone (Algorithm 1 needs no counts).
inline unsigned seg_grid(int cap) { return (unsigned)max(1, min(cap, 2048)); }

}  // namespace

hipError_t launch_seg_gather(const eaas_segment* segs, const int32_t* num_tokens, int n_seg,
                             int cap, int H, int k, const int32_t* id_off, int e_local,
                             uint16_t* x_cat, int32_t* ids_cat, float* w_cat,
                             hipStream_t stream) {
  hipLaunchKernelGGL(seg_gather_kernel, dim3(seg_grid(cap)), dim3(kSegThreads), 0, stream, segs,
                     num_tokens, n_seg, cap, H, k, id_off, e_local, x_cat, ids_cat, w_cat);
  return hipGetLastError();
}

hipError_t launch_slot_snapshot(const eaas_slot* slots, int n_slots, int cap, int n_layers,
                                int e_layer, eaas_segment* segs, int32_t* num_tokens,
                                int32_t* id_off, int32_t* taken, hipStream_t stream) {
  hipLaunchKernelGGL(slot_snapshot_kernel, dim3(1), dim3(kMaxSegments), 0, stream, slots,
                     n_slots, cap, n_layers, e_layer, segs, num_tokens, id_off, taken);
  return hipGetLastError();
}

hipError_t launch_slot_complete(const eaas_slot* slots, int n_slots, const int32_t* taken,
                                hipStream_t stream) {
  hipLaunchKernelGGL(slot_complete_kernel, dim3(1), dim3(kMaxSegments), 0, stream, slots,
                     n_slots, taken);
  return hipGetLastError();
}

hipError_t launch_seg_combine(const eaas_segment* segs, const int32_t* num_tokens, int n_seg,
                              int cap, int H, int k, const float* stage, const int32_t* inv,
                              const float* w, bool out_fp32, hipStream_t stream) {
  if (out_fp32)
    hipLaunchKernelGGL((seg_combine_kernel<true>), dim3(seg_grid(cap)), dim3(kSegThreads), 0,
                       stream, segs, num_tokens, n_seg, cap, H, k, stage, inv, w);
  else
    hipLaunchKernelGGL((seg_combine_kernel<false>), dim3(seg_grid(cap)), dim3(kSegThreads), 0,
                       stream, segs, num_tokens, n_seg, cap, H, k, stage, inv, w);
  return hipGetLastError();
}

}  // namespace eaas
