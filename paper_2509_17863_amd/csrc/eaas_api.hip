// C ABI of the expert-server forward step: host-side validation, workspace
// layout and kernel enqueueing.  No allocation, no synchronisation, no
// device-to-host traffic: every entry point only enqueues work on `stream`.
#include <limits.h>
#include <stdint.h>

#include <algorithm>
#include <atomic>
#include <mutex>

#include "common.h"
#include "internal.h"

namespace {

using namespace eaas;

constexpr size_t kAlign = 256;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

struct WsLayout {
  size_t hist, counts, offsets, perm, inv, active, h, stage, total;
  // fp8 activations: h held as hq [R,I] + hs [R,I/128] inside the h region,
  // x quantized into xq [T,H] + xs [T,H/128] after it
  size_t hq, hs, xq, xs;
  // bytes eaas_route_permute uses (the histogram) and eaas_expert_ffn_grouped
  // uses (everything before the staging); the forward uses `total`
  size_t route_total, ffn_total;
  // dynamic batch only: the requests gathered into one contiguous batch
  size_t x_cat, ids_cat, w_cat, seg_total;
};

WsLayout layout(const eaas_shape& s, int w_dtype = EAAS_BF16) {
  const size_t R = (size_t)s.T * s.k;
  WsLayout L{};
  size_t o = 0;
  L.hist = o;    o = align_up(o + (size_t)route_blocks((int)R) * s.E * 4);
  L.route_total = o;
  L.counts = o;  o = align_up(o + (size_t)s.E * 4);
  L.offsets = o; o = align_up(o + (size_t)(s.E + 1) * 4);
  L.perm = o;    o = align_up(o + R * 4);
  L.inv = o;     o = align_up(o + R * 4);
  L.active = o;  o = align_up(o + (size_t)(s.E + 1) * 4);
  L.h = o;
  L.hq = L.h;
  L.hs = align_up(L.h + R * s.I);
  o = align_up(std::max(L.h + R * s.I * 2, L.hs + R * (s.I / 128) * 4));
  if (w_dtype == EAAS_FP8_E4M3_A8) {
    L.xq = o;    o = align_up(o + (size_t)s.T * s.H);
    L.xs = o;    o = align_up(o + (size_t)s.T * (s.H / 128) * 4);
  }
  L.ffn_total = o;
  L.stage = o;   o = align_up(o + R * s.H * 4);
  L.total = o;
  L.x_cat = o;   o = align_up(o + (size_t)s.T * s.H * 2);
  L.ids_cat = o; o = align_up(o + R * 4);
  L.w_cat = o;   o = align_up(o + R * 4);
  L.seg_total = o;
  return L;
}

int check_shape(const eaas_shape* s) {
  if (!s) return EAAS_ERR_INVALID_ARG;
  if (s->T < 0 || s->H <= 0 || s->I <= 0 || s->E <= 0 || s->k <= 0) return EAAS_ERR_INVALID_ARG;
  if (s->H % 128 || s->I % 128 || s->E > kMaxExperts || s->k > kMaxTopK) return EAAS_ERR_UNSUPPORTED;
  const long long R = (long long)s->T * s->k;
  // 32-bit element offsets inside the kernels
  if (R > INT_MAX || (long long)s->T * s->H > INT_MAX || R * s->I > INT_MAX ||
      4LL * s->I * s->H > INT_MAX)
    return EAAS_ERR_UNSUPPORTED;
  return EAAS_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

bool routing_ok(const eaas_routing* r) {
  return r && r->counts && r->offsets && r->perm && r->inv && r->active &&
         aligned16(r->perm) && aligned16(r->inv);
}

bool weights_ok(const void* wgu, const float* sgu, const void* wd, const float* sd, int w_dtype) {
  if (!wgu || !wd || !aligned16(wgu) || !aligned16(wd)) return false;
  if (w_dtype == EAAS_BF16) return true;
  if (w_dtype == EAAS_FP8_E4M3 || w_dtype == EAAS_FP8_E4M3_A8 || w_dtype == EAAS_FP8_E4M3_TILED)
    return sgu && sd;
  return false;
}

// Shape limits of a weight dtype beyond check_shape (fp8 activations and
// tiled fp8 weights: the down projection's N = H in 256-wide tiles).
int check_dtype_shape(const eaas_shape* s, int w_dtype) {
  if ((w_dtype == EAAS_FP8_E4M3_A8 || w_dtype == EAAS_FP8_E4M3_TILED) && s->H % 256)
    return EAAS_ERR_UNSUPPORTED;
  return EAAS_OK;
}

bool known_wdtype(int w_dtype) {
  return w_dtype == EAAS_BF16 || w_dtype == EAAS_FP8_E4M3 || w_dtype == EAAS_FP8_E4M3_A8 ||
         w_dtype == EAAS_FP8_E4M3_TILED;
}

// FfnArgs members of the weight dtype (h and y are set by the caller).
void set_dtype_args(FfnArgs& a, int w_dtype, char* base, const WsLayout& L) {
  a.fp8 = w_dtype == EAAS_FP8_E4M3 || w_dtype == EAAS_FP8_E4M3_A8 ||
          w_dtype == EAAS_FP8_E4M3_TILED;
  a.act8 = w_dtype == EAAS_FP8_E4M3_A8;
  a.tiled = w_dtype == EAAS_FP8_E4M3_TILED;
  if (a.act8) {
    a.xq = reinterpret_cast<const uint8_t*>(base + L.xq);
    a.xs = reinterpret_cast<const float*>(base + L.xs);
    a.hq = reinterpret_cast<uint8_t*>(base + L.hq);
    a.hs = reinterpret_cast<float*>(base + L.hs);
  }
}

// fp8 activations: quantize x into the workspace before the gate/up GEMM.
hipError_t quantize_x(const FfnArgs& a, char* base, const WsLayout& L, hipStream_t hs) {
  if (!a.act8) return hipSuccess;
  return launch_quantize_rows(a.x, a.T, a.H, reinterpret_cast<uint8_t*>(base + L.xq),
                              reinterpret_cast<float*>(base + L.xs), hs);
}

int hip_status(hipError_t e) { return e == hipSuccess ? EAAS_OK : EAAS_ERR_HIP; }

eaas_routing ws_routing(char* base, const WsLayout& L) {
  eaas_routing r;
  r.counts = reinterpret_cast<int32_t*>(base + L.counts);
  r.offsets = reinterpret_cast<int32_t*>(base + L.offsets);
  r.perm = reinterpret_cast<int32_t*>(base + L.perm);
  r.inv = reinterpret_cast<int32_t*>(base + L.inv);
  r.active = reinterpret_cast<int32_t*>(base + L.active);
  return r;
}

}  // namespace

extern "C" {

size_t eaas_workspace_bytes(const eaas_shape* s, int w_dtype) {
  if (check_shape(s) != EAAS_OK) return 0;
  if (!known_wdtype(w_dtype)) return 0;
  if (check_dtype_shape(s, w_dtype) != EAAS_OK) return 0;
  return layout(*s, w_dtype).total;
}

size_t eaas_workspace_bytes_for(const eaas_shape* s, int w_dtype, int entry) {
  if (eaas_workspace_bytes(s, w_dtype) == 0) return 0;
  const WsLayout L = layout(*s, w_dtype);
  switch (entry) {
    case EAAS_ENTRY_ROUTE_PERMUTE: return L.route_total;
    case EAAS_ENTRY_FFN_GROUPED: return L.ffn_total;
    case EAAS_ENTRY_FORWARD: return L.total;
    default: return 0;
  }
}

int eaas_workspace_region(const eaas_shape* s, int w_dtype, int region, size_t* offset,
                          size_t* bytes) {
  if (!offset || !bytes) return EAAS_ERR_INVALID_ARG;
  if (eaas_workspace_bytes(s, w_dtype) == 0) return EAAS_ERR_UNSUPPORTED;
  const WsLayout L = layout(*s, w_dtype);
  const size_t R = (size_t)s->T * s->k;
  const bool a8 = w_dtype == EAAS_FP8_E4M3_A8;
  switch (region) {
    case EAAS_WS_H:
      if (a8) return EAAS_ERR_INVALID_ARG;
      *offset = L.h; *bytes = R * s->I * 2; return EAAS_OK;
    case EAAS_WS_HQ:
      if (!a8) return EAAS_ERR_INVALID_ARG;
      *offset = L.hq; *bytes = R * s->I; return EAAS_OK;
    case EAAS_WS_HS:
      if (!a8) return EAAS_ERR_INVALID_ARG;
      *offset = L.hs; *bytes = R * (s->I / 128) * 4; return EAAS_OK;
    case EAAS_WS_XQ:
      if (!a8) return EAAS_ERR_INVALID_ARG;
      *offset = L.xq; *bytes = (size_t)s->T * s->H; return EAAS_OK;
    case EAAS_WS_XS:
      if (!a8) return EAAS_ERR_INVALID_ARG;
      *offset = L.xs; *bytes = (size_t)s->T * (s->H / 128) * 4; return EAAS_OK;
    case EAAS_WS_STAGE:
      *offset = L.stage; *bytes = R * s->H * 4; return EAAS_OK;
    default:
      return EAAS_ERR_INVALID_ARG;
  }
}

int eaas_tile_weights_fp8(const eaas_shape* s, int which, const void* w, void* w_tiled,
                          void* stream) {
  int st = check_shape(s);
  if (st != EAAS_OK) return st;
  if (which != EAAS_GATE_UP && which != EAAS_DOWN) return EAAS_ERR_INVALID_ARG;
  if ((st = check_dtype_shape(s, EAAS_FP8_E4M3_TILED)) != EAAS_OK) return st;
  if (!w || !w_tiled || !aligned16(w) || !aligned16(w_tiled)) return EAAS_ERR_INVALID_ARG;
  const int N = which == EAAS_GATE_UP ? 2 * s->I : s->H;
  const int K = which == EAAS_GATE_UP ? s->H : s->I;
  const size_t bytes = (size_t)s->E * N * K;
  const uintptr_t a = (uintptr_t)w, b = (uintptr_t)w_tiled;
  if (a < b + bytes && b < a + bytes) return EAAS_ERR_INVALID_ARG;  // no overlap, no in-place
  return hip_status(launch_tile_weights_fp8(static_cast<const uint8_t*>(w),
                                            static_cast<uint8_t*>(w_tiled), s->E, N, K,
                                            which == EAAS_GATE_UP ? s->I : 0,
                                            reinterpret_cast<hipStream_t>(stream)));
}

int eaas_quantize_rows_fp8(const void* x, int64_t rows, int32_t K, void* q, float* s,
                           void* stream) {
  if (rows < 0 || K <= 0) return EAAS_ERR_INVALID_ARG;
  if (K % 128 || rows * (int64_t)K > INT_MAX) return EAAS_ERR_UNSUPPORTED;
  if (rows == 0) return EAAS_OK;
  if (!x || !q || !s || !aligned16(x) || !aligned16(q)) return EAAS_ERR_INVALID_ARG;
  return hip_status(launch_quantize_rows(static_cast<const uint16_t*>(x), rows, K,
                                         static_cast<uint8_t*>(q), s,
                                         reinterpret_cast<hipStream_t>(stream)));
}

int eaas_route_permute(const eaas_shape* s, const int32_t* topk_ids, const eaas_routing* r,
                       void* ws, size_t ws_bytes, void* stream) {
  int st = check_shape(s);
  if (st != EAAS_OK) return st;
  if (s->T == 0) return EAAS_OK;
  if (!topk_ids || !routing_ok(r)) return EAAS_ERR_INVALID_ARG;
  const WsLayout L = layout(*s);
  if (!ws || !aligned16(ws) || ws_bytes < L.route_total) return EAAS_ERR_WORKSPACE;
  char* base = static_cast<char*>(ws);
  return hip_status(launch_route_permute(topk_ids, s->T * s->k, s->E, *r,
                                         reinterpret_cast<int32_t*>(base + L.hist),
                                         reinterpret_cast<hipStream_t>(stream)));
}

int eaas_expert_ffn_grouped(const eaas_shape* s, const void* x, const eaas_routing* r,
                            const void* w_gate_up, const float* w_gate_up_scale,
                            const void* w_down, const float* w_down_scale, int w_dtype,
                            float* y_perm, void* ws, size_t ws_bytes, void* stream) {
  int st = check_shape(s);
  if (st != EAAS_OK) return st;
  if (s->T == 0) return EAAS_OK;
  if (!x || !aligned16(x) || !routing_ok(r) || !y_perm || !aligned16(y_perm) ||
      !weights_ok(w_gate_up, w_gate_up_scale, w_down, w_down_scale, w_dtype))
    return EAAS_ERR_INVALID_ARG;
  if ((st = check_dtype_shape(s, w_dtype)) != EAAS_OK) return st;
  const WsLayout L = layout(*s, w_dtype);
  if (!ws || !aligned16(ws) || ws_bytes < L.ffn_total) return EAAS_ERR_WORKSPACE;
  char* base = static_cast<char*>(ws);
  FfnArgs a{};
  a.T = s->T; a.H = s->H; a.I = s->I; a.E = s->E; a.k = s->k;
  a.x = static_cast<const uint16_t*>(x);
  a.perm = r->perm;
  a.offsets = r->offsets;
  a.active = r->active;
  a.w_gate_up = w_gate_up;
  a.s_gate_up = w_gate_up_scale;
  a.w_down = w_down;
  a.s_down = w_down_scale;
  set_dtype_args(a, w_dtype, base, L);
  a.h = reinterpret_cast<uint16_t*>(base + L.h);
  a.y = y_perm;
  a.epilogue = kDownPlain;
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = quantize_x(a, base, L, hs);
  if (e == hipSuccess) e = launch_gate_up(a, hs);
  if (e == hipSuccess) e = launch_down(a, hs);
  return hip_status(e);
}

int eaas_unpermute_combine(const eaas_shape* s, const float* y_perm, const eaas_routing* r,
                           const float* topk_weights, void* out, int out_dtype, void* stream) {
  int st = check_shape(s);
  if (st != EAAS_OK) return st;
  if (s->T == 0) return EAAS_OK;
  if (!y_perm || !aligned16(y_perm) || !routing_ok(r) || !topk_weights || !out ||
      !aligned16(out) || (out_dtype != EAAS_BF16 && out_dtype != EAAS_FP32))
    return EAAS_ERR_INVALID_ARG;
  return hip_status(launch_combine(y_perm, r->inv, topk_weights, s->T, s->H, s->k, false, out,
                                   out_dtype == EAAS_FP32, reinterpret_cast<hipStream_t>(stream)));
}

int eaas_expert_forward_profiled(const eaas_shape* s, const void* x, const int32_t* topk_ids,
                                 const float* topk_weights, const void* w_gate_up,
                                 const float* w_gate_up_scale, const void* w_down,
                                 const float* w_down_scale, int w_dtype, void* out,
                                 int out_dtype, const eaas_routing* r, void* ws,
                                 size_t ws_bytes, void* stream, void* const* events) {
  int st = check_shape(s);
  if (st != EAAS_OK) return st;
  if (s->T == 0) return EAAS_OK;
  if (!x || !aligned16(x) || !topk_ids || !topk_weights || !out || !aligned16(out) ||
      (out_dtype != EAAS_BF16 && out_dtype != EAAS_FP32) ||
      !weights_ok(w_gate_up, w_gate_up_scale, w_down, w_down_scale, w_dtype) ||
      (r && !routing_ok(r)))
    return EAAS_ERR_INVALID_ARG;
  // out may alias x exactly (bf16 write-back into the payload), nothing else
  const size_t xb = (size_t)s->T * s->H * 2;
  const size_t ob = (size_t)s->T * s->H * (out_dtype == EAAS_FP32 ? 4 : 2);
  const uintptr_t xp = (uintptr_t)x, op = (uintptr_t)out;
  if (op == xp) {
    if (out_dtype != EAAS_BF16) return EAAS_ERR_INVALID_ARG;
  } else if (op < xp + xb && xp < op + ob) {
    return EAAS_ERR_INVALID_ARG;
  }
  if ((st = check_dtype_shape(s, w_dtype)) != EAAS_OK) return st;
  const WsLayout L = layout(*s, w_dtype);
  if (!ws || !aligned16(ws) || ws_bytes < L.total) return EAAS_ERR_WORKSPACE;
  char* base = static_cast<char*>(ws);
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  const eaas_routing rt = r ? *r : ws_routing(base, L);
  auto mark = [&](int i) -> hipError_t {
    if (!events || !events[i]) return hipSuccess;
    return hipEventRecord(reinterpret_cast<hipEvent_t>(events[i]), hs);
  };
  if (mark(0) != hipSuccess) return EAAS_ERR_HIP;
  hipError_t e = launch_route_permute(topk_ids, s->T * s->k, s->E, rt,
                                      reinterpret_cast<int32_t*>(base + L.hist), hs);
  if (e != hipSuccess) return EAAS_ERR_HIP;
  float* stage = reinterpret_cast<float*>(base + L.stage);
  FfnArgs a{};
  a.T = s->T; a.H = s->H; a.I = s->I; a.E = s->E; a.k = s->k;
  a.x = static_cast<const uint16_t*>(x);
  a.perm = rt.perm;
  a.offsets = rt.offsets;
  a.active = rt.active;
  a.w_gate_up = w_gate_up;
  a.s_gate_up = w_gate_up_scale;
  a.w_down = w_down;
  a.s_down = w_down_scale;
  set_dtype_args(a, w_dtype, base, L);
  a.h = reinterpret_cast<uint16_t*>(base + L.h);
  a.y = stage;
  a.epilogue = kDownBySlot;
  // (fp8 activations: x is quantized in the routing interval, so the gate/up
  // interval times the GEMM alone)
  e = quantize_x(a, base, L, hs);
  if (e != hipSuccess || mark(1) != hipSuccess) return EAAS_ERR_HIP;
  e = launch_gate_up(a, hs);
  if (e != hipSuccess || mark(2) != hipSuccess) return EAAS_ERR_HIP;
  e = launch_down(a, hs);
  if (e != hipSuccess || mark(3) != hipSuccess) return EAAS_ERR_HIP;
  e = launch_combine(stage, rt.inv, topk_weights, s->T, s->H, s->k, true, out,
                     out_dtype == EAAS_FP32, hs);
  if (e != hipSuccess || mark(4) != hipSuccess) return EAAS_ERR_HIP;
  return EAAS_OK;
}

int eaas_expert_forward(const eaas_shape* s, const void* x, const int32_t* topk_ids,
                        const float* topk_weights, const void* w_gate_up,
                        const float* w_gate_up_scale, const void* w_down,
                        const float* w_down_scale, int w_dtype, void* out, int out_dtype,
                        const eaas_routing* r, void* ws, size_t ws_bytes, void* stream) {
  return eaas_expert_forward_profiled(s, x, topk_ids, topk_weights, w_gate_up, w_gate_up_scale,
                                      w_down, w_down_scale, w_dtype, out, out_dtype, r, ws,
                                      ws_bytes, stream, nullptr);
}

size_t eaas_segments_workspace_bytes(const eaas_shape* s, int w_dtype) {
  if (eaas_workspace_bytes(s, w_dtype) == 0) return 0;
  return layout(*s, w_dtype).seg_total;
}

int eaas_expert_forward_segments(const eaas_shape* s, const eaas_segment* segs,
                                 const int32_t* num_tokens, int n_seg, const void* w_gate_up,
                                 const float* w_gate_up_scale, const void* w_down,
                                 const float* w_down_scale, int w_dtype, int out_dtype, void* ws,
                                 size_t ws_bytes, void* stream) {
  int st = check_shape(s);
  if (st != EAAS_OK) return st;
  if (n_seg < 0 || n_seg > kMaxSegments) return EAAS_ERR_INVALID_ARG;
  if ((st = check_dtype_shape(s, w_dtype)) != EAAS_OK) return st;
  if (s->T == 0 || n_seg == 0) return EAAS_OK;
  if (!segs || !num_tokens || (out_dtype != EAAS_BF16 && out_dtype != EAAS_FP32) ||
      !weights_ok(w_gate_up, w_gate_up_scale, w_down, w_down_scale, w_dtype))
    return EAAS_ERR_INVALID_ARG;
  const WsLayout L = layout(*s, w_dtype);
  if (!ws || !aligned16(ws) || ws_bytes < L.seg_total) return EAAS_ERR_WORKSPACE;
  char* base = static_cast<char*>(ws);
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  const int cap = s->T;
  uint16_t* x_cat = reinterpret_cast<uint16_t*>(base + L.x_cat);
  int32_t* ids_cat = reinterpret_cast<int32_t*>(base + L.ids_cat);
  float* w_cat = reinterpret_cast<float*>(base + L.w_cat);
  hipError_t e = launch_seg_gather(segs, num_tokens, n_seg, cap, s->H, s->k, nullptr, s->E,
                                   x_cat, ids_cat, w_cat, hs);
  if (e != hipSuccess) return EAAS_ERR_HIP;
  const eaas_routing rt = ws_routing(base, L);
  e = launch_route_permute(ids_cat, cap * s->k, s->E, rt,
                           reinterpret_cast<int32_t*>(base + L.hist), hs);
  if (e != hipSuccess) return EAAS_ERR_HIP;
  float* stage = reinterpret_cast<float*>(base + L.stage);
  FfnArgs a{};
  a.T = cap; a.H = s->H; a.I = s->I; a.E = s->E; a.k = s->k;
  a.x = x_cat;
  a.perm = rt.perm;
  a.offsets = rt.offsets;
  a.active = rt.active;
  a.w_gate_up = w_gate_up;
  a.s_gate_up = w_gate_up_scale;
  a.w_down = w_down;
  a.s_down = w_down_scale;
  set_dtype_args(a, w_dtype, base, L);
  a.h = reinterpret_cast<uint16_t*>(base + L.h);
  a.y = stage;
  a.epilogue = kDownBySlot;
  e = quantize_x(a, base, L, hs);
  if (e == hipSuccess) e = launch_gate_up(a, hs);
  if (e == hipSuccess) e = launch_down(a, hs);
  if (e == hipSuccess)
    e = launch_seg_combine(segs, num_tokens, n_seg, cap, s->H, s->k, stage, rt.inv, w_cat,
                           out_dtype == EAAS_FP32, hs);
  return hip_status(e);
}

}  // extern "C"

namespace {

// Server-step extras after the dynamic-batch layout: the request records of
// the taken slots, their counts, layer group offsets and the taken mask.
struct SlotLayout {
  size_t segs, counts, id_off, taken, total;
};

SlotLayout slot_layout(size_t seg_total) {
  SlotLayout S{};
  size_t o = seg_total;
  S.segs = o;   o = align_up(o + (size_t)kMaxSegments * sizeof(eaas_segment));
  S.counts = o; o = align_up(o + (size_t)kMaxSegments * 4);
  S.id_off = o; o = align_up(o + (size_t)kMaxSegments * 4);
  S.taken = o;  o = align_up(o + (size_t)kMaxSegments * 4);
  S.total = o;
  return S;
}

// The step's shape over all layers: one group per (layer, expert).
int server_shape(const eaas_shape* s, int n_layers, eaas_shape* g) {
  int st = check_shape(s);
  if (st != EAAS_OK) return st;
  if (n_layers < 1) return EAAS_ERR_INVALID_ARG;
  if ((long long)n_layers * s->E > kMaxExperts) return EAAS_ERR_UNSUPPORTED;
  *g = *s;
  g->E = n_layers * s->E;
  return check_shape(g);
}

}  // namespace

extern "C" {

size_t eaas_server_workspace_bytes(const eaas_shape* s, int n_layers, int w_dtype) {
  eaas_shape g;
  if (server_shape(s, n_layers, &g) != EAAS_OK) return 0;
  if (eaas_workspace_bytes(&g, w_dtype) == 0) return 0;
  return slot_layout(layout(g, w_dtype).seg_total).total;
}

int eaas_server_step(const eaas_shape* s, const eaas_slot* slots, int n_slots,
                     const eaas_layer_weights* layers, int n_layers, int w_dtype, void* ws,
                     size_t ws_bytes, void* stream) {
  eaas_shape g;
  int st = server_shape(s, n_layers, &g);
  if (st != EAAS_OK) return st;
  if (n_slots < 0 || n_slots > kMaxSegments) return EAAS_ERR_INVALID_ARG;
  if ((st = check_dtype_shape(&g, w_dtype)) != EAAS_OK) return st;
  if (n_slots == 0) return EAAS_OK;
  if (!slots || !layers ||
      !known_wdtype(w_dtype))
    return EAAS_ERR_INVALID_ARG;
  const WsLayout L = layout(g, w_dtype);
  const SlotLayout SL = slot_layout(L.seg_total);
  if (!ws || !aligned16(ws) || ws_bytes < SL.total) return EAAS_ERR_WORKSPACE;
  char* base = static_cast<char*>(ws);
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  const int cap = s->T;
  eaas_segment* segs = reinterpret_cast<eaas_segment*>(base + SL.segs);
  int32_t* counts = reinterpret_cast<int32_t*>(base + SL.counts);
  int32_t* id_off = reinterpret_cast<int32_t*>(base + SL.id_off);
  int32_t* taken = reinterpret_cast<int32_t*>(base + SL.taken);
  hipError_t e = launch_slot_snapshot(slots, n_slots, cap, n_layers, s->E, segs, counts, id_off,
                                      taken, hs);
  if (e != hipSuccess) return EAAS_ERR_HIP;
  if (cap > 0) {
    uint16_t* x_cat = reinterpret_cast<uint16_t*>(base + L.x_cat);
    int32_t* ids_cat = reinterpret_cast<int32_t*>(base + L.ids_cat);
    float* w_cat = reinterpret_cast<float*>(base + L.w_cat);
    e = launch_seg_gather(segs, counts, n_slots, cap, g.H, g.k, id_off, s->E, x_cat, ids_cat,
                          w_cat, hs);
    if (e != hipSuccess) return EAAS_ERR_HIP;
    const eaas_routing rt = ws_routing(base, L);
    e = launch_route_permute(ids_cat, cap * g.k, g.E, rt,
                             reinterpret_cast<int32_t*>(base + L.hist), hs);
    if (e != hipSuccess) return EAAS_ERR_HIP;
    FfnArgs a{};
    a.T = cap; a.H = g.H; a.I = g.I; a.E = g.E; a.k = g.k;
    a.x = x_cat;
    a.perm = rt.perm;
    a.offsets = rt.offsets;
    a.active = rt.active;
    set_dtype_args(a, w_dtype, base, L);
    a.h = reinterpret_cast<uint16_t*>(base + L.h);
    a.y = reinterpret_cast<float*>(base + L.stage);
    a.epilogue = kDownBySlot;
    a.layers = layers;
    a.e_layer = s->E;
    e = quantize_x(a, base, L, hs);
    if (e == hipSuccess) e = launch_gate_up(a, hs);
    if (e == hipSuccess) e = launch_down(a, hs);
    if (e == hipSuccess)
      e = launch_seg_combine(segs, counts, n_slots, cap, g.H, g.k, a.y, rt.inv, w_cat, false, hs);
    if (e != hipSuccess) return EAAS_ERR_HIP;
  }
  return hip_status(launch_slot_complete(slots, n_slots, taken, hs));
}

}  // extern "C"

namespace {

// Library-owned scratch of the allocation-free forward: static device memory,
// one copy per GPU the library is loaded on.  In host code `scratch` only
// names the symbol; its device address is taken once per device with
// hipGetSymbolAddress and used from then on.
static __device__ __align__(256) char scratch[EAAS_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

// The scratch array's address on the current device (hipGetSymbolAddress on
// the first call there, with that device current; cached afterwards).
int scratch_on_current_device(void** ptr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return EAAS_ERR_HIP;
  void* p = g_scratch[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch[dev].load(std::memory_order_relaxed);
    if (!p) {
      if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return EAAS_ERR_HIP;
      g_scratch[dev].store(p, std::memory_order_release);
    }
  }
  *ptr = p;
  return EAAS_OK;
}

}  // namespace

extern "C" {

int eaas_expert_forward_noalloc(const eaas_shape* s, const void* x, const int32_t* topk_ids,
                                const float* topk_weights, const void* w_gate_up,
                                const float* w_gate_up_scale, const void* w_down,
                                const float* w_down_scale, int w_dtype, void* out, int out_dtype,
                                const eaas_routing* r, void* stream) {
  int st = check_shape(s);
  if (st != EAAS_OK) return st;
  if (s->T == 0) return EAAS_OK;
  const size_t need = eaas_workspace_bytes(s, w_dtype);
  if (need == 0) return check_dtype_shape(s, w_dtype) != EAAS_OK ? EAAS_ERR_UNSUPPORTED
                                                                  : EAAS_ERR_INVALID_ARG;
  if (need > (size_t)EAAS_NOALLOC_SCRATCH_BYTES) return EAAS_ERR_WORKSPACE;
  void* ws = nullptr;
  if ((st = scratch_on_current_device(&ws)) != EAAS_OK) return st;
  return eaas_expert_forward_profiled(s, x, topk_ids, topk_weights, w_gate_up, w_gate_up_scale,
                                      w_down, w_down_scale, w_dtype, out, out_dtype, r, ws,
                                      (size_t)EAAS_NOALLOC_SCRATCH_BYTES, stream, nullptr);
}

const char* eaas_status_string(int status) {
  switch (status) {
    case EAAS_OK: return "ok";
    case EAAS_ERR_INVALID_ARG: return "invalid argument";
    case EAAS_ERR_UNSUPPORTED: return "unsupported shape";
    case EAAS_ERR_WORKSPACE: return "workspace missing or too small";
    case EAAS_ERR_HIP: return "HIP launch error";
    default: return "unknown status";
  }
}

}  // extern "C"
