// Weighted sum of expert outputs back into token order (EaaS §3.3: the server
// writes the weighted sum of expert outputs into the request's payload; the
// weights are the router scores carried in the payload, §3.2).
//
// out[t, :] = sum over ascending j of valid slots s = t*k + j of w[s] * Y_s,
// accumulated in fp32 from +0 with every product and sum rounded separately
// (contraction into fused multiply-add is switched off in the kernel), so the
// result does not depend on which entry point produced Y_s:
//   rows_by_slot: Y_s at row s (the fused step: the down projection's
//                 epilogue stores each row at its slot)
//   otherwise:    Y_s at row inv[s] (modular entry point, permuted order)
// One workgroup per (token, 1024-column block); each thread owns 4
// consecutive columns, and the staged rows are read once (non-temporal).
#include "common.h"
#include "internal.h"

namespace eaas {
namespace {

constexpr int kCombineThreads = 256;
constexpr int kCombineCols = kCombineThreads * 4;  // columns per workgroup

// One slot's staged row: at row s (BY_SLOT) or at row inv[s].
template <bool BY_SLOT>
__device__ __forceinline__ f32x4 load_slot(const float* __restrict__ y, int s, int row, int H,
                                           int c) {
  if (BY_SLOT)
    return __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(y + (size_t)s * H + c));
  return *reinterpret_cast<const f32x4*>(y + (size_t)row * H + c);
}

// grid: (T, ceil(H / kCombineCols)); each thread owns 4 consecutive columns.
// KU > 0 (k <= KU): the k rows and weights are all requested before the
// first add, so a thread has k loads in flight; the adds still run in
// ascending j.
template <bool BY_SLOT, bool OUT_FP32, int KU>
__global__ __launch_bounds__(kCombineThreads) void combine_kernel(
    const float* __restrict__ y, const int32_t* __restrict__ inv,
    const float* __restrict__ w, int T, int H, int k, void* __restrict__ out) {
  // products and sums are rounded separately: no fused multiply-add here
#pragma clang fp contract(off)
  const int t = blockIdx.x;
  const int c = blockIdx.y * kCombineCols + threadIdx.x * 4;
  if (c >= H) return;
  f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  auto add = [&](const f32x4& v, float wj) {
#pragma clang fp contract(off)
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[q] = acc[q] + wj * v[q];
  };
  if constexpr (KU > 0) {
    f32x4 v[KU];
    float wv[KU];
    bool live[KU];
#pragma unroll
    for (int j = 0; j < KU; ++j) {
      const int s = t * k + j;
      const int row = j < k ? inv[s] : -1;
      live[j] = row >= 0 && row < T * k;
      v[j] = live[j] ? load_slot<BY_SLOT>(y, s, row, H, c) : f32x4{};
      wv[j] = live[j] ? w[s] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < KU; ++j)
      if (live[j]) add(v[j], wv[j]);
  } else {
    for (int j = 0; j < k; ++j) {
      const int s = t * k + j;
      const int row = inv[s];
      if (row < 0 || row >= T * k) continue;
      add(load_slot<BY_SLOT>(y, s, row, H, c), w[s]);
    }
  }
  if (OUT_FP32) {
    *reinterpret_cast<f32x4*>(static_cast<float*>(out) + (size_t)t * H + c) = acc;
  } else {
    u32x2 o;
    o[0] = pack_bf16x2(acc[0], acc[1]);
    o[1] = pack_bf16x2(acc[2], acc[3]);
    *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(out) + (size_t)t * H + c) = o;
  }
}

template <bool BY_SLOT, bool OUT_FP32>
void launch_combine_k(dim3 grid, dim3 block, hipStream_t stream, const float* y,
                      const int32_t* inv, const float* w, int T, int H, int k, void* out) {
  if (k <= 8)
    hipLaunchKernelGGL((combine_kernel<BY_SLOT, OUT_FP32, 8>), grid, block, 0, stream, y, inv, w,
                       T, H, k, out);
  else
    hipLaunchKernelGGL((combine_kernel<BY_SLOT, OUT_FP32, 0>), grid, block, 0, stream, y, inv, w,
                       T, H, k, out);
}

}  // namespace

hipError_t launch_combine(const float* y, const int32_t* inv, const float* w,
                          int T, int H, int k, bool by_slot, void* out,
                          bool out_fp32, hipStream_t stream) {
  if (T <= 0) return hipSuccess;
  const dim3 grid(T, (H + kCombineCols - 1) / kCombineCols), block(kCombineThreads);
  if (by_slot) {
    if (out_fp32) launch_combine_k<true, true>(grid, block, stream, y, inv, w, T, H, k, out);
    else launch_combine_k<true, false>(grid, block, stream, y, inv, w, T, H, k, out);
  } else {
    if (out_fp32) launch_combine_k<false, true>(grid, block, stream, y, inv, w, T, H, k, out);
    else launch_combine_k<false, false>(grid, block, stream, y, inv, w, T, H, k, out);
  }
  return hipGetLastError();
}

}  // namespace eaas
