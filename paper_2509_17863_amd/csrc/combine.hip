// Weighted sum of expert outputs back into token order (EaaS §3.3: the server
// writes the weighted sum of expert outputs into the request's payload; the
// weights are the router scores carried in the payload, §3.2).
//
// out[t, :] = sum over ascending j of valid slots s = t*k + j of w[s] * Y_s,
// accumulated in fp32 from +0 with every product and sum rounded separately
// (contraction into fused multiply-add is switched off in the kernel), so the
// result does not depend on which entry point produced Y_s:
//   rows_by_slot_weighted: y holds w[s] * Y_s already, at row s (fused step)
//   otherwise:             y holds Y at row inv[s] (modular entry point)
// One workgroup per token row; each thread owns 4 consecutive columns per
// step, so the k rows (contiguous in the fused layout) stream coalesced.
#include "common.h"
#include "internal.h"

namespace eaas {
namespace {

constexpr int kCombineThreads = 256;

template <bool BY_SLOT, bool OUT_FP32>
__global__ __launch_bounds__(kCombineThreads) void combine_kernel(
    const float* __restrict__ y, const int32_t* __restrict__ inv,
    const float* __restrict__ w, int T, int H, int k, void* __restrict__ out) {
  // products and sums are rounded separately: no fused multiply-add here
#pragma clang fp contract(off)
  const int t = blockIdx.x;
  __shared__ int s_row[kMaxTopK];
  __shared__ float s_w[kMaxTopK];
  if (threadIdx.x < k) {
    const int s = t * k + threadIdx.x;
    s_row[threadIdx.x] = inv[s];
    s_w[threadIdx.x] = w[s];
  }
  __syncthreads();
  const int h4 = H / 4;
  for (int c = threadIdx.x; c < h4; c += kCombineThreads) {
    f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int j = 0; j < k; ++j) {
      const int row = s_row[j];
      if (row < 0 || row >= T * k) continue;
      if (BY_SLOT) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(y + (size_t)(t * k + j) * H + 4 * c);
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[q] = acc[q] + v[q];
      } else {
        const f32x4 v = *reinterpret_cast<const f32x4*>(y + (size_t)row * H + 4 * c);
        const float wj = s_w[j];
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[q] = acc[q] + wj * v[q];
      }
    }
    if (OUT_FP32) {
      *reinterpret_cast<f32x4*>(static_cast<float*>(out) + (size_t)t * H + 4 * c) = acc;
    } else {
      u32x2 o;
      o[0] = pack_bf16x2(acc[0], acc[1]);
      o[1] = pack_bf16x2(acc[2], acc[3]);
      *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(out) + (size_t)t * H + 4 * c) = o;
    }
  }
}

}  // namespace

hipError_t launch_combine(const float* y, const int32_t* inv, const float* w,
                          int T, int H, int k, bool by_slot, void* out,
                          bool out_fp32, hipStream_t stream) {
  if (T <= 0) return hipSuccess;
  const dim3 grid(T), block(kCombineThreads);
  if (by_slot) {
    if (out_fp32) hipLaunchKernelGGL((combine_kernel<true, true>), grid, block, 0, stream, y, inv, w, T, H, k, out);
    else hipLaunchKernelGGL((combine_kernel<true, false>), grid, block, 0, stream, y, inv, w, T, H, k, out);
  } else {
    if (out_fp32) hipLaunchKernelGGL((combine_kernel<false, true>), grid, block, 0, stream, y, inv, w, T, H, k, out);
    else hipLaunchKernelGGL((combine_kernel<false, false>), grid, block, 0, stream, y, inv, w, T, H, k, out);
  }
  return hipGetLastError();
}

}  // namespace eaas
