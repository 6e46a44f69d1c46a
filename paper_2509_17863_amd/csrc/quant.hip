// Activation quantization for the fp8-weight, fp8-activation step: per row
// and per block of 128 channels, s = amax / 448 (1 for an all-zero block)
// and q = e4m3fn(x / s), rounded to nearest even and saturated at 448.  The
// scale and the quotient are correctly rounded fp32, so the codes are the
// ones a plain fp32 evaluation of that definition gives.  (The paper's
// grouped-GEMM engine, §4.1, consumes block-scaled fp8 operands; the
// blocking follows the weights' 128-channel K blocks.)
#include "common.h"
#include "internal.h"

namespace eaas {
namespace {

constexpr int kQuantThreads = 256;

// One lane: 8 consecutive values (16 bytes of bf16); 16 lanes: one block of
// 128.  Blocks never straddle rows (K is a multiple of 128), and the chunk
// count is a multiple of 16, so a 16-lane group is always wholly active.
__global__ __launch_bounds__(kQuantThreads) void quantize_rows_kernel(
    const uint16_t* __restrict__ x, long long n_chunks, uint8_t* __restrict__ q,
    float* __restrict__ s) {
  for (long long c = (long long)blockIdx.x * kQuantThreads + threadIdx.x; c < n_chunks;
       c += (long long)gridDim.x * kQuantThreads) {
    const u32x4 raw = *reinterpret_cast<const u32x4*>(x + c * 8);
    float v[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(raw[i] << 16);
      v[2 * i + 1] = __uint_as_float(raw[i] & 0xffff0000u);
    }
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) amax = fmaxf(amax, fabsf(v[i]));
#pragma unroll
    for (int m = 8; m >= 1; m >>= 1) amax = fmaxf(amax, __shfl_xor(amax, m, 16));
    const float sc = amax > 0.0f ? amax / 448.0f : 1.0f;
    u32x2 o;
    o[0] = pack_e4m3x4(v[0] / sc, v[1] / sc, v[2] / sc, v[3] / sc);
    o[1] = pack_e4m3x4(v[4] / sc, v[5] / sc, v[6] / sc, v[7] / sc);
    *reinterpret_cast<u32x2*>(q + c * 8) = o;
    if ((c & 15) == 0) s[c >> 4] = sc;
  }
}

}  // namespace

hipError_t launch_quantize_rows(const uint16_t* x, long long rows, int K, uint8_t* q, float* s,
                                hipStream_t stream) {
  const long long n_chunks = rows * (K / 8);
  if (n_chunks <= 0) return hipSuccess;
  const long long blocks = (n_chunks + kQuantThreads - 1) / kQuantThreads;
  const unsigned grid = (unsigned)(blocks < 8192 ? blocks : 8192);
  hipLaunchKernelGGL(quantize_rows_kernel, dim3(grid), dim3(kQuantThreads), 0, stream, x,
                     n_chunks, q, s);
  return hipGetLastError();
}

}  // namespace eaas
