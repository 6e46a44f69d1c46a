/*
 * eaas.h -- C ABI of one stateless expert server's forward step on gfx950.
 *
 * The operation (EaaS, §3.3 "Asynchronous Server Operation", and Fig. 5): the
 * server takes a batch of ready requests, reorganises the tokens by expert,
 * runs the grouped expert computation, and writes back for every token the
 * weighted sum of its experts' outputs.  The request payload (§3.2 "Data
 * Payload") carries the hidden states, an expert id per token slot and the
 * router score used for weighting; the header carries the batch size (§3.2
 * "Header").  The server is stateless (§2.4, §3.3): nothing survives between
 * calls, so every call is a pure function of its arguments.
 *
 * Symbols: T tokens (header batch_size), H hidden size, I expert intermediate
 * size, E resident experts on this server, k expert slots per token,
 * R = T*k slots.  Slot s = t*k + j.  A slot is valid iff 0 <= topk_ids[s] < E;
 * other ids (experts hosted by other servers) are skipped, not errors.
 *
 * Expert FFN (the paper names only "expert computations"; this library
 * implements the SwiGLU form without bias):
 *     y_e(x) = W_down[e] . ( silu(W_gate[e] . x) * (W_up[e] . x) )
 * with W_gate_up[e] = [W_gate[e]; W_up[e]] stacked by rows (gate rows [0,I),
 * up rows [I,2I)), W_gate_up[E,2I,H] and W_down[E,H,I], both [out,in]
 * row-major.  Accumulation is fp32; the intermediate h is rounded once to
 * bf16 (round to nearest even); the weighted sum is fp32, summed over valid
 * slots in ascending j starting from +0.
 *
 * Weights are bf16, or OCP fp8 e4m3fn with one fp32 scale per 128x128 block
 * of each expert matrix (W = q * s): scale arrays [E,2I/128,H/128] and
 * [E,H/128,I/128], row-major.
 *
 * Conventions for every entry point:
 *   - All array pointers are DEVICE pointers owned by the caller; the shape
 *     descriptor and the routing descriptor themselves live in host memory.
 *   - The library never allocates, frees or synchronises.  Scratch memory is
 *     the caller's workspace `ws` of at least eaas_workspace_bytes() bytes,
 *     256-byte aligned.  Its contents are undefined between calls.
 *   - `stream` is a hipStream_t passed as void* (NULL = null stream).  All work
 *     is enqueued on it with no host synchronisation and no device-to-host
 *     readback, so calls can be captured in a hipGraph.
 *   - Arguments are validated on the host before anything is enqueued; on any
 *     error a negative status is returned and nothing is enqueued.  T = 0 is
 *     a valid empty batch: EAAS_OK, nothing enqueued, outputs left untouched
 *     (pointers may then be NULL).  Device arrays must be 16-byte aligned
 *     (EAAS_ERR_INVALID_ARG otherwise).
 *   - Calls are re-entrant; concurrent calls must use distinct workspaces and
 *     outputs.
 *   - NaN and Inf in the data propagate; they are not errors.
 */
#ifndef EAAS_H
#define EAAS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct eaas_shape {
  int32_t T; /* tokens in the batch (>= 0)                              */
  int32_t H; /* hidden size, multiple of 128                             */
  int32_t I; /* expert intermediate size, multiple of 128                */
  int32_t E; /* resident experts, 1..1024                                */
  int32_t k; /* slots per token, 1..64                                   */
} eaas_shape;

enum eaas_status {
  EAAS_OK = 0,
  EAAS_ERR_INVALID_ARG = -1, /* null pointer, negative size, bad dtype, overlap
                                (k > E is valid: see eaas_route_permute) */
  EAAS_ERR_UNSUPPORTED = -2, /* H or I not a multiple of 128, E > 1024, k > 64,
                                or past the 32-bit element offsets the kernels
                                use: T*k, T*H, T*k*I or 4*I*H above 2^31 - 1 */
  EAAS_ERR_WORKSPACE = -3,   /* ws NULL, misaligned or smaller than the entry
                                point's eaas_workspace_bytes_for */
  EAAS_ERR_HIP = -4          /* a kernel launch was rejected by the runtime  */
};

enum eaas_dtype {
  EAAS_BF16 = 0,     /* bfloat16 bit patterns (uint16)                    */
  EAAS_FP8_E4M3 = 1, /* OCP fp8 e4m3fn bit patterns (uint8), weights only */
  EAAS_FP32 = 2,     /* IEEE binary32, outputs only                       */
  /* As a weight dtype: fp8 e4m3fn weights (as EAAS_FP8_E4M3) and fp8
   * activations.  The step quantizes x per token and h per row, per block of
   * 128 channels (s = amax/448, 1 for an all-zero block; q = e4m3(a/s),
   * nearest even, saturating at 448; fp32 arithmetic), and runs both grouped
   * GEMMs on fp8 x fp8 MFMAs with fp32 accumulation, scaling each 128-wide K
   * block's partial sums by its row scale times its weight block scale (the
   * block-scaled fp8 GEMM of the grouped-GEMM engine named in §4.1).  Needs
   * H a multiple of 256.  Accepted by every entry point that takes a
   * weight dtype. */
  EAAS_FP8_E4M3_A8 = 3,
  /* As a weight dtype: the fp8 e4m3fn weights of EAAS_FP8_E4M3 (same values,
   * same scales, same results bit for bit) stored in the tiled layout that
   * eaas_tile_weights_fp8 writes, which the decode-sized fp8 GEMMs stream as
   * contiguous blocks instead of rows K bytes apart.  Needs H a multiple of
   * 256.  Accepted by every entry point that takes a weight dtype. */
  EAAS_FP8_E4M3_TILED = 4
};

/*
 * Routing of a batch: the token reorganisation of §3.3 plus the compacted
 * active-expert list of the group-shrink prefix scan (§4.1).  Device arrays:
 *   counts [E]    valid slots per expert
 *   offsets[E+1]  exclusive prefix sum of counts; offsets[E] = valid slots
 *   perm   [R]    row r -> slot s; rows are grouped by expert in ascending
 *                 expert id and, inside an expert, in ascending slot order
 *                 (the unique stable counting sort); rows >= offsets[E] hold -1
 *   inv    [R]    slot s -> row, or -1 for an invalid slot
 *   active [E+1]  active[0] = number of experts with counts > 0, then those
 *                 experts in ascending order, then zeros
 */
typedef struct eaas_routing {
  int32_t *counts;
  int32_t *offsets;
  int32_t *perm;
  int32_t *inv;
  int32_t *active;
} eaas_routing;

/* Bytes of workspace that every entry point below accepts for this shape and
 * weight dtype (the maximum over the entry points).  Returns 0 for a shape the
 * library rejects. */
size_t eaas_workspace_bytes(const eaas_shape *s, int w_dtype);

/* Bytes of workspace one entry point needs for this shape and weight dtype:
 *   EAAS_ENTRY_ROUTE_PERMUTE  eaas_route_permute (its histogram only; w_dtype
 *                             is ignored beyond validation)
 *   EAAS_ENTRY_FFN_GROUPED    eaas_expert_ffn_grouped (h, and for
 *                             EAAS_FP8_E4M3_A8 the quantized x; no staging)
 *   EAAS_ENTRY_FORWARD        eaas_expert_forward(_profiled), which is
 *                             eaas_workspace_bytes
 * Each is at most eaas_workspace_bytes(s, w_dtype).  Returns 0 for a shape or
 * dtype the library rejects and for an unknown entry. */
enum eaas_entry {
  EAAS_ENTRY_ROUTE_PERMUTE = 0, EAAS_ENTRY_FFN_GROUPED = 1, EAAS_ENTRY_FORWARD = 2
};
size_t eaas_workspace_bytes_for(const eaas_shape *s, int w_dtype, int entry);

/* Where a forward call leaves its intermediates inside the workspace (for
 * inspection and tests; the contents are those of the last call that used
 * the workspace, rows in the grouped order of the routing):
 *   EAAS_WS_H      h [R,I] bf16 (bf16 and fp8-weight modes)
 *   EAAS_WS_HQ     h quantized [R,I] e4m3fn codes   (EAAS_FP8_E4M3_A8)
 *   EAAS_WS_HS     its scales [R,I/128] fp32         (EAAS_FP8_E4M3_A8)
 *   EAAS_WS_XQ     x quantized [T,H] e4m3fn codes    (EAAS_FP8_E4M3_A8)
 *   EAAS_WS_XS     its scales [T,H/128] fp32         (EAAS_FP8_E4M3_A8)
 *   EAAS_WS_STAGE  expert outputs [R,H] fp32 (not yet weighted), row = slot
 *                  t*k+j (eaas_expert_forward; invalid slots untouched)
 * Writes the byte offset and size of the region.  Returns INVALID_ARG for a
 * null output pointer, an unknown region or one the dtype does not have,
 * UNSUPPORTED for a shape or dtype eaas_workspace_bytes rejects. */
enum eaas_ws_region {
  EAAS_WS_H = 0, EAAS_WS_HQ = 1, EAAS_WS_HS = 2, EAAS_WS_XQ = 3, EAAS_WS_XS = 4,
  EAAS_WS_STAGE = 5
};
int eaas_workspace_region(const eaas_shape *s, int w_dtype, int region, size_t *offset,
                          size_t *bytes);

/* Activation quantization of the EAAS_FP8_E4M3_A8 step, on its own:
 *   x [rows,K] bf16 (device), K a multiple of 128 and rows*K < 2^31
 *   q [rows,K] e4m3fn codes (device, written), s [rows,K/128] fp32 (device,
 *   written): per row and block of 128 channels, s = amax/448 (1 if the block
 *   is all zero), q = e4m3fn(x/s) rounded to nearest even and saturated at
 *   +-448, with s and x/s correctly rounded fp32.
 * x, q 16-byte aligned.  rows == 0 is a no-op.  Errors: INVALID_ARG (null or
 * misaligned pointer, rows < 0, K <= 0), UNSUPPORTED (K % 128, size), HIP. */
int eaas_quantize_rows_fp8(const void *x, int64_t rows, int32_t K, void *q, float *s,
                           void *stream);

/* The fp8 weight layout of EAAS_FP8_E4M3_TILED (weights stay resident on a
 * server, so they are rearranged once, when loaded).
 *   which    EAAS_GATE_UP: w is W_gate_up [E,2I,H] (N = 2I rows, K = H);
 *            EAAS_DOWN:    w is W_down    [E,H,I] (N = H rows, K = I)
 *   w        e4m3fn codes [E,N,K], row-major (device, read)
 *   w_tiled  E*N*K bytes (device, written), the same codes reordered: with
 *            BN = 512 for a gate/up matrix whose 2I is a multiple of 512 and
 *            256 otherwise, for expert e, N tile tn < N/BN, K tile kt < K/64,
 *            j < BN and b < 64,
 *              w_tiled[((e*(N/BN) + tn)*(K/64) + kt)*BN*64 + j*64 + b]
 *                = w[e][row(tn, j)][64*kt + b],
 *            row(tn, j) = tn*BN + j for W_down; for W_gate_up the tile's BN/2
 *            gate rows come first: row(tn, j) = tn*BN/2 + j for j < BN/2,
 *            I + tn*BN/2 + j - BN/2 otherwise.
 * The block scales are not moved.  s->T is not used (any valid value).
 * Errors: INVALID_ARG (unknown `which`, null, misaligned or overlapping
 * pointers), UNSUPPORTED (the shape, or H not a multiple of 256), HIP. */
enum eaas_matrix { EAAS_GATE_UP = 0, EAAS_DOWN = 1 };
int eaas_tile_weights_fp8(const eaas_shape *s, int which, const void *w, void *w_tiled,
                          void *stream);

/* Token reorganisation + group-shrink (§3.3 Fig. 5, §4.1).
 *   topk_ids [T,k] int32   expert id per slot (payload `expert_id`, §3.2)
 *   r                      all five arrays written, bit-exact and deterministic
 * Needs ws of eaas_workspace_bytes_for(s, EAAS_BF16, EAAS_ENTRY_ROUTE_PERMUTE)
 * bytes (a histogram of ceil(T*k/2048) x E ints); H and I only need to pass
 * validation.  k may exceed E: slots whose ids name other servers' experts are
 * skipped, so a server with fewer experts than a token has slots is valid. */
int eaas_route_permute(const eaas_shape *s, const int32_t *topk_ids,
                       const eaas_routing *r, void *ws, size_t ws_bytes,
                       void *stream);

/* Grouped expert FFN over the reorganised rows (§3.3 "grouped GEMM").
 *   x          [T,H] bf16 hidden states (payload, §3.2)
 *   r          routing produced by eaas_route_permute for the same ids
 *   w_gate_up  [E,2I,H] bf16 or fp8; w_gate_up_scale [E,2I/128,H/128] fp32
 *              for fp8, ignored (may be NULL) for bf16
 *   w_down     [E,H,I]  bf16 or fp8; w_down_scale [E,H/128,I/128] likewise
 *   y_perm     [R,H] fp32 output: row r = y_{e(r)}(x[perm[r]/k]), unweighted;
 *              rows >= offsets[E] are left untouched
 * Only experts listed in r->active are read.  Needs ws of
 * eaas_workspace_bytes_for(s, w_dtype, EAAS_ENTRY_FFN_GROUPED) bytes. */
int eaas_expert_ffn_grouped(const eaas_shape *s, const void *x,
                            const eaas_routing *r, const void *w_gate_up,
                            const float *w_gate_up_scale, const void *w_down,
                            const float *w_down_scale, int w_dtype,
                            float *y_perm, void *ws, size_t ws_bytes,
                            void *stream);

/* Weighted sum of expert outputs back into token order (§3.3 "the weighted sum
 * of expert outputs", weights = router_score of §3.2).
 *   out[t,:] = sum over ascending j with valid slot t*k+j of
 *              fp32(topk_weights[t,j] * y_perm[inv[t*k+j],:]), from +0
 *   out        [T,H] bf16 (round to nearest even of the fp32 sum) or fp32;
 *              tokens with no valid slot get zeros. */
int eaas_unpermute_combine(const eaas_shape *s, const float *y_perm,
                           const eaas_routing *r, const float *topk_weights,
                           void *out, int out_dtype, void *stream);

/* The whole step: route_permute, grouped FFN and weighted combine in one call,
 * result bitwise equal to calling the three entry points above in sequence.
 *   r      optional (NULL: routing lives in the workspace); when given it is
 *          written as by eaas_route_permute
 *   out    [T,H] bf16 or fp32.  out == x (exactly, bf16 out) is allowed: the
 *          result is written back into the request payload in place (§3.3);
 *          any other overlap of out with x is EAAS_ERR_INVALID_ARG. */
int eaas_expert_forward(const eaas_shape *s, const void *x,
                        const int32_t *topk_ids, const float *topk_weights,
                        const void *w_gate_up, const float *w_gate_up_scale,
                        const void *w_down, const float *w_down_scale,
                        int w_dtype, void *out, int out_dtype,
                        const eaas_routing *r, void *ws, size_t ws_bytes,
                        void *stream);

/* eaas_expert_forward, plus timing marks for measurement: events[0..4] are
 * hipEvent_t handles (passed as void*, NULL entries skipped) recorded on
 * `stream` before routing, before the gate/up GEMM, before the down GEMM,
 * before the combine and after it.  events itself may be NULL.  Same kernels,
 * same results as eaas_expert_forward. */
int eaas_expert_forward_profiled(const eaas_shape *s, const void *x,
                                 const int32_t *topk_ids,
                                 const float *topk_weights,
                                 const void *w_gate_up,
                                 const float *w_gate_up_scale,
                                 const void *w_down, const float *w_down_scale,
                                 int w_dtype, void *out, int out_dtype,
                                 const eaas_routing *r, void *ws,
                                 size_t ws_bytes, void *stream,
                                 void *const *events);

/*
 * Dynamic batch of several clients' requests (§3.3: the server aggregates the
 * ready requests of its clients into one batch and writes each client's
 * results back into that client's payload; §3.2: a buffer slot's payload and
 * its header's batch size).
 *
 * One request, as laid out in a client's buffer slot (device pointers,
 * 16-byte aligned; only the first num_tokens[b] rows belong to the request):
 *   x            [n,H] bf16 hidden states
 *   topk_ids     [n,k] int32 expert ids (ids outside [0,E) are skipped)
 *   topk_weights [n,k] fp32 router scores
 *   out          [n,H] weighted sums, bf16 or fp32 per out_dtype.  out == x
 *                (bf16) writes the result back into the payload in place; out
 *                must not overlap any other request's arrays.
 */
typedef struct eaas_segment {
  const void *x;
  const int32_t *topk_ids;
  const float *topk_weights;
  void *out;
} eaas_segment;

/* Workspace bytes of eaas_expert_forward_segments for a capacity of s->T
 * tokens (0 for a shape the library rejects). */
size_t eaas_segments_workspace_bytes(const eaas_shape *s, int w_dtype);

/* The step on a dynamic batch of requests whose token counts are read on the
 * device, so the same call (or a captured graph of it) serves any mix of
 * batch sizes.  The tokens are walked with Algorithm 1 of §4 (a static grid
 * over requests of varying length that skips empty ones).
 *   s->T        capacity: grids and workspace are sized for at most s->T
 *               tokens in all requests together
 *   segs        [n_seg] eaas_segment, a DEVICE array
 *   num_tokens  [n_seg] int32, a DEVICE array: request b's batch size (header
 *               batch_size).  0 means no request from that client this step;
 *               negative counts count as 0.  Requests are batched in slot
 *               order; tokens past the capacity are not processed and their
 *               out rows are left untouched.
 *   n_seg       0..1024 (0: nothing enqueued)
 * For every request b, out rows [0, num_tokens[b]) receive exactly what
 * eaas_expert_forward writes for those tokens when run on the requests
 * concatenated in slot order; no other memory of the requests is written. */
int eaas_expert_forward_segments(const eaas_shape *s, const eaas_segment *segs,
                                 const int32_t *num_tokens, int n_seg,
                                 const void *w_gate_up,
                                 const float *w_gate_up_scale,
                                 const void *w_down, const float *w_down_scale,
                                 int w_dtype, int out_dtype, void *ws,
                                 size_t ws_bytes, void *stream);

/*
 * One server step over the clients' buffer slots (§3.2 "Shared Communication
 * Buffer Design", §3.3 "Asynchronous Server Operation", §3.4 offline clients).
 *
 * Every client owns one slot on the server, in device memory:
 *   flag      slot state, one of the eaas_slot_state values; the paper uses
 *             one byte, here it is a 32-bit word so that host and device can
 *             update it with naturally aligned atomic accesses
 *   header    [2] int32: layer_id, batch_size
 *   x         [capacity,H] bf16 hidden states; the step overwrites rows
 *             [0, n) with the request's weighted sums (the results are written
 *             back into the data payload, §3.3)
 *   topk_ids, topk_weights  [capacity,k] int32 / fp32 (payload, §3.2)
 * A server may hold several layers: layers[L] holds the weights of layer L
 * (the arrays and dtype of eaas_expert_forward), and requests of different
 * layers are batched into one grouped step (expert e of layer L is group
 * L*E + e).
 */
enum eaas_slot_state {
  EAAS_SLOT_EMPTY = 0,   /* the client may write a request                   */
  EAAS_SLOT_READY = 1,   /* client write done: the server may take it         */
  EAAS_SLOT_DONE = 2,    /* server computation done: the client may read      */
  EAAS_SLOT_OFFLINE = 3  /* client reported offline: the server leaves it alone */
};

typedef struct eaas_slot {
  int32_t *flag;
  const int32_t *header;
  void *x;
  const int32_t *topk_ids;
  const float *topk_weights;
  int64_t capacity;
} eaas_slot;

typedef struct eaas_layer_weights {
  const void *w_gate_up;
  const float *w_gate_up_scale;
  const void *w_down;
  const float *w_down_scale;
} eaas_layer_weights;

/* Workspace bytes of eaas_server_step (0 for a shape the library rejects). */
size_t eaas_server_workspace_bytes(const eaas_shape *s, int n_layers, int w_dtype);

/* One server step: snapshot the slot flags, take the ready slots (flag 1) in
 * slot order while their batch sizes (clamped to [0, capacity]) fit the step
 * capacity s->T, run them as one dynamic batch, write each request's weighted
 * sums (bf16) over its hidden states, then set the taken slots' flags to 2.
 *   s->E        experts per layer; n_layers * s->E <= 1024
 *   slots       [n_slots] eaas_slot, a DEVICE array; n_slots 0..1024
 *   layers      [n_layers] eaas_layer_weights, a DEVICE array, all of w_dtype
 * Slots in any other state, ready slots that do not fit (they stay ready for a
 * later step), and payload rows past a request are not written.  A taken
 * request whose layer_id names no layer of this server gets zeros.  Within a
 * taken request, every row equals eaas_expert_forward on the requests of its
 * layer concatenated in slot order.  The flags are written after all results,
 * behind a system-scope fence.  Two steps over the same slots must not
 * overlap in time (a later step runs on the same stream or after the first). */
int eaas_server_step(const eaas_shape *s, const eaas_slot *slots, int n_slots,
                     const eaas_layer_weights *layers, int n_layers, int w_dtype,
                     void *ws, size_t ws_bytes, void *stream);

/*
 * For callers that cannot allocate device memory: code under hipGraph capture,
 * tight serving loops, harnesses that forbid hipMalloc.  eaas_expert_forward
 * with the caller's workspace replaced by a library-owned device array of
 * EAAS_NOALLOC_SCRATCH_BYTES bytes per GPU: static device memory that every
 * GPU the library is loaded on holds until the process ends.  The call itself
 * allocates and frees nothing.
 *   Same arguments and results as eaas_expert_forward (bitwise), without
 *   ws / ws_bytes.  The array used is that of the device current at the call
 *   (hipGetDevice), which must be the device `stream` belongs to.
 *   A shape that needs more, eaas_workspace_bytes(s, w_dtype) >
 *   EAAS_NOALLOC_SCRATCH_BYTES (80 MiB: it holds the 256-token, H 7168, I 2048,
 *   32-expert, top-8 decode step with fp8 or bf16 weights), returns
 *   EAAS_ERR_WORKSPACE and enqueues nothing; other errors as in
 *   eaas_expert_forward.
 *   Every call on one GPU shares that GPU's array, which keeps the last
 *   call's intermediates (each call rebuilds everything it reads, so nothing
 *   has to start at zero).  Calls that overlap in time on one GPU (on
 *   different streams, or from several host threads) race on the array and
 *   give undefined results: serialise them, e.g. on one stream.
 */
#define EAAS_NOALLOC_SCRATCH_BYTES (80u << 20)
int eaas_expert_forward_noalloc(const eaas_shape *s, const void *x,
                                const int32_t *topk_ids,
                                const float *topk_weights,
                                const void *w_gate_up,
                                const float *w_gate_up_scale,
                                const void *w_down, const float *w_down_scale,
                                int w_dtype, void *out, int out_dtype,
                                const eaas_routing *r, void *stream);

/* Static, human-readable name of a status code. */
const char *eaas_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* EAAS_H */
