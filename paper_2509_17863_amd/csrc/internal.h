// Host-side launchers shared between the C ABI and the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/eaas.h"

namespace eaas {

// Slots handled by one workgroup of the histogram and scatter kernels.
constexpr int kRouteChunk = 2048;

// Requests in one dynamic batch (their token counts sit in shared memory).
constexpr int kMaxSegments = 1024;

inline int route_blocks(int R) { return (R + kRouteChunk - 1) / kRouteChunk; }

// Enqueue the three routing kernels.  `hist` holds route_blocks(R) * E ints.
hipError_t launch_route_permute(const int32_t* ids, int R, int E,
                                const eaas_routing& r, int32_t* hist,
                                hipStream_t stream);

// Which epilogue the down projection uses.
enum DownEpilogue {
  kDownPlain = 0,   // y[r, :] = Y[r, :] (rows in permuted order)
  kDownBySlot = 1,  // y[perm[r], :] = Y[r, :] (rows by slot; the combine weights them)
};

struct FfnArgs {
  int T, H, I, E, k;
  const uint16_t* x;          // [T,H] bf16
  const int32_t* perm;        // [R]
  const int32_t* offsets;     // [E+1]
  const int32_t* active;      // [E+1]
  const void* w_gate_up;      // [E,2I,H]
  const float* s_gate_up;     // [E,2I/128,H/128] (fp8 only)
  const void* w_down;         // [E,H,I]
  const float* s_down;        // [E,H/128,I/128] (fp8 only)
  bool fp8;
  uint16_t* h;                // [R,I] bf16 scratch
  float* y;                   // [R,H] fp32
  int epilogue;               // DownEpilogue
  // server step over several layers: E = layers x e_layer groups whose weights
  // come from the per-layer records (w_* and s_* above are then unused)
  const eaas_layer_weights* layers = nullptr;
  int e_layer = 0;
  // fp8 activations (with fp8 weights): x and h quantized per row and 128
  // channels; h is then held only as hq / hs
  bool act8 = false;
  const uint8_t* xq = nullptr;  // [T,H]
  const float* xs = nullptr;    // [T,H/128]
  uint8_t* hq = nullptr;        // [R,I]
  float* hs = nullptr;          // [R,I/128]
  // fp8 weights stored in the tiled layout of launch_tile_weights_fp8
  bool tiled = false;
};

// x [rows,K] bf16 -> q [rows,K] e4m3fn and s [rows,K/128]: per row and 128
// channels, s = amax/448 (1 if all zero), q = e4m3(x/s) (nearest even,
// saturating).
hipError_t launch_quantize_rows(const uint16_t* x, long long rows, int K, uint8_t* q, float* s,
                                hipStream_t stream);

// fp8 weights [E,N,K] -> the tiled layout the fp8-weight ring kernels read
// (weight stages contiguous).  I > 0: a gate/up matrix (N = 2I, gate rows then
// up rows); I == 0: a down matrix.
hipError_t launch_tile_weights_fp8(const uint8_t* w, uint8_t* out, int E, int N, int K, int I,
                                   hipStream_t stream);

// Gate/up GEMM with the SiLU*mul epilogue into h.
hipError_t launch_gate_up(const FfnArgs& a, hipStream_t stream);
// Down GEMM from h into y (epilogue per a.epilogue).
hipError_t launch_down(const FfnArgs& a, hipStream_t stream);

// out[t] = sum_j w[s] * y[by_slot ? s : inv[s]] over valid slots s = t*k+j.
hipError_t launch_combine(const float* y, const int32_t* inv, const float* w,
                          int T, int H, int k, bool rows_by_slot,
                          void* out, bool out_fp32, hipStream_t stream);

// Dynamic batch (Algorithm 1 walks): gather the requests' tokens into the
// contiguous batch of `cap` rows (slots of unused capacity get id -1), and
// write each request's weighted sums of the by-slot fp32 staging rows.
// id_off (optional): per request, the group offset of its ids (valid ids are
// those in [0, e_local)); a negative offset masks the request's slots.
hipError_t launch_seg_gather(const eaas_segment* segs, const int32_t* num_tokens, int n_seg,
                             int cap, int H, int k, const int32_t* id_off, int e_local,
                             uint16_t* x_cat, int32_t* ids_cat, float* w_cat,
                             hipStream_t stream);
hipError_t launch_seg_combine(const eaas_segment* segs, const int32_t* num_tokens, int n_seg,
                              int cap, int H, int k, const float* stage, const int32_t* inv,
                              const float* w, bool out_fp32, hipStream_t stream);

// Server step: snapshot the slots into a dynamic batch (records, counts,
// layer group offsets, taken mask), and mark the taken slots done.
hipError_t launch_slot_snapshot(const eaas_slot* slots, int n_slots, int cap, int n_layers,
                                int e_layer, eaas_segment* segs, int32_t* num_tokens,
                                int32_t* id_off, int32_t* taken, hipStream_t stream);
hipError_t launch_slot_complete(const eaas_slot* slots, int n_slots, const int32_t* taken,
                                hipStream_t stream);

}  // namespace eaas
