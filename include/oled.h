/*
 * oled.h - C ABI of the OLED-MoE block-MoE layer hot path for MI355X (gfx950).
 *
 * One MoE layer l in one denoising iteration i of a semi-autoregressive dLLM,
 * run with a fixed-capacity per-layer GPU expert cache (OLED-MoE, Sec. 4.1):
 *
 *   route_block        the gate's routed expert ids and gate scores for every
 *                      token of the block (Sec. 4.1), plus the expert
 *                      histogram, offsets and stable token permutation
 *   moe_forward_cached the SwiGLU experts that are cached (hits, A & R) run
 *                      directly on the GPU (Sec. 4.1); enqueued without
 *                      waiting for the routing result on the host
 *   apply_misses       misses M = A \ R of the layer (Sec. 4.2): every miss
 *                      is transferred host->device into a staging slot (G = M)
 *                      and computed on the GPU once it has landed
 *   score_and_retain   reuse priorities p_e (the priority equation of
 *                      Sec. 4.3, psi(c) = c; stale residents score zero) and
 *                      the retention rule R' = Top_C(R u G, p) of Sec. 4.2;
 *                      after a forward, in the same launch as the
 *                      gate-weighted combine of all k routes of every token
 *
 * Call order per (layer, iteration): route_block -> [moe_forward_cached] ->
 * apply_misses -> score_and_retain. Exactly one layer is in flight per
 * context; any other order returns OLED_ERR_STATE and changes nothing.
 * moe_forward_cached may be skipped (control path only: apply_misses then
 * only transfers); the cache state does not depend on expert outputs. The
 * layer output y is complete once the work score_and_retain enqueued has run.
 *
 * The cache state (resident sets, slot tables, free slots) lives in device
 * memory and only the library's kernels change it, in stream order: the
 * routing kernel gives every miss a free staging slot, the retention kernel
 * commits. The transfer of the misses (oled_config.copy_mode):
 *  OLED_COPY_SHADER  workgroups of the hit experts' GEMM launches copy the
 *                    staged misses' weights from the pinned pool over PCIe
 *                    while the other workgroups compute; no call of a layer
 *                    waits for the device unless a report is asked for.
 *  OLED_COPY_SDMA    apply_misses waits for the routing result and copies the
 *                    misses with hipMemcpyAsync on a copy stream; the miss
 *                    GEMMs are launched once the host has seen the copies land.
 * Counts of a layer (hits, misses, bytes) are in the pinned routing records;
 * apply_misses with a report, oled_read_layer_state and oled_collect_stats
 * read them.
 *
 * Conventions
 *  - Every function returns an oled_status and never aborts. Host-detected
 *    errors (OLED_ERR_INVALID_ARG, OLED_ERR_STATE, OLED_ERR_UNSUPPORTED) leave
 *    all host and device state unchanged. oled_last_error() describes the last
 *    failure of a context.
 *  - "_dev" pointers are device memory on the context's GPU, "host" pointers
 *    are host memory. Streams are hipStream_t passed as void* (NULL = the null
 *    stream). The caller keeps every buffer it passes alive until the stream
 *    work that reads it has completed.
 *  - Layouts are row-major and dense. Token t of the block is row t.
 *  - One host thread per context. The four calls of a layer must use the same
 *    compute stream; a new stream at route_block is ordered after the old one.
 *  - Routing indices, permutations, hit/miss counts and retained sets are
 *    deterministic integers; layer outputs are bitwise identical for any cache
 *    residency (the cache only changes where weights are read from).
 */
#ifndef OLED_H_
#define OLED_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  OLED_OK = 0,
  OLED_ERR_INVALID_ARG = 1,  /* bad argument, or bad data found on the device */
  OLED_ERR_OUT_OF_MEMORY = 2,
  OLED_ERR_HIP = 3,          /* a HIP runtime call failed */
  OLED_ERR_STATE = 4,        /* call out of order for this context */
  OLED_ERR_UNSUPPORTED = 5   /* shape outside the supported range */
} oled_status;

typedef enum { OLED_F32 = 0, OLED_BF16 = 1 } oled_dtype;

/* How the misses reach their staging slots (see above). */
typedef enum { OLED_COPY_SHADER = 0, OLED_COPY_SDMA = 1 } oled_copy_mode;

/* Retention key of score_and_retain. OLED_POLICY_PRIORITY is the paper's
 * confidence-gate priority (Sec. 4.3); LRU and LFU are the comparison
 * policies of its evaluation (Sec. 5.1, Sec. 5.3), ranking the same
 * candidates by the layer iteration of each expert's last activation, or by
 * the routes sent to it so far, with the same tie-breaks. */
typedef enum { OLED_POLICY_PRIORITY = 0, OLED_POLICY_LRU = 1, OLED_POLICY_LFU = 2 } oled_policy;


/*
 * Shape and resources of one MoE layer stack.
 *  hidden H, inter I: multiples of 128. n_experts E in [1, 256]. top_k k in
 *  [1, min(E, 16)]. n_layers L >= 1. capacity C >= 0 experts per layer (C = 0:
 *  every active expert misses; C >= E: full residency); with adapt_period > 0
 *  the layers share C_total = L * min(C, E) and each holds at most E. max_tokens Tmax in
 *  [1, 65535] (bounds the integer priority sums, see score_and_retain).
 *  dtype: activations, weights and outputs; accumulation is fp32.
 *
 *  host_pool: caller-owned pinned host memory (hipHostMalloc, oled_host_alloc
 *  or a pinned torch tensor) of host_pool_blocks expert blocks, each
 *  3*H*I*elem bytes in the packed layout written by oled_pack_expert.
 *  host_block_of[l*E + e] in [0, host_pool_blocks) names the block of expert
 *  e of layer l; several experts may share one block. The pool must outlive
 *  the context; the table is copied at creation. The pool must be mapped for
 *  device access (hipHostMalloc memory is).
 */
typedef struct {
  int32_t hidden;
  int32_t inter;
  int32_t n_experts;
  int32_t top_k;
  int32_t n_layers;
  int32_t capacity;
  int32_t max_tokens;
  int32_t dtype;            /* oled_dtype */
  int32_t device;           /* HIP device ordinal */
  int32_t profile_ops;      /* bit (1 << oled_op_kind) set: time that operation with HIP
                               events on its stream (oled_profile_collect); 0: off */
  const void* host_pool;
  int64_t host_pool_blocks;
  const int64_t* host_block_of;
  int32_t copy_mode;        /* oled_copy_mode */
  int32_t adapt_period;     /* 0: every layer keeps capacity min(C, E). > 0: layer-adaptive
                               cache sizing (Sec. 4.3) after every adapt_period-th completed
                               iteration of the layer stack (the paper uses 5); see
                               score_and_retain. Needs n_layers <= 1024. */
  int32_t policy;           /* oled_policy */
  int32_t coop;             /* 1: cooperative compensation (Sec. 4.4): misses are split
                               between transfer and CPU execution by apply_misses_coop.
                               Needs OLED_COPY_SHADER. */
  int32_t coop_threads;     /* host threads of the CPU expert execution (>= 1 with coop) */
  int32_t reserved;
  double coop_t_h2d_us;     /* T_H2D: transfer time of one expert (profiled, microseconds) */
  double coop_tau_cpu_us;   /* tau_CPU: CPU time of one expert for one token (microseconds) */
  double coop_nbar;         /* nbar: average routed tokens per missed expert (profiled) */
  double coop_lambda_us;    /* lambda: weight of the transferred priority mass in J, in
                               microseconds per unit of priority (p summed over G) */
} oled_config;

/* Result of apply_misses for the layer (Sec. 4.2). Counts are experts. */
typedef struct {
  int32_t n_active;       /* |A| */
  int32_t n_hits;         /* |A & R| */
  int32_t n_misses;       /* |M| = |A \ R|, all transferred */
  int32_t n_resident;     /* |R| before execution */
  int32_t rejected_layer; /* a layer whose last retention was rejected for an
                             invalid confidence since the previous report, else -1 */
  int32_t n_cpu;          /* misses executed on the CPU (apply_misses_coop), else 0 */
  int64_t h2d_bytes;      /* bytes transferred host->device for the misses */
} oled_miss_report;

/* Totals over the routing calls since the last oled_collect_stats. */
typedef struct {
  int64_t layer_iters;    /* route_block calls */
  int64_t n_active;       /* sum of |A| */
  int64_t n_hits;         /* sum of |A & R| */
  int64_t n_misses;       /* sum of |M| */
  int64_t n_transferred;  /* misses given a staging slot and transferred */
  int64_t h2d_bytes;      /* their bytes */
  int64_t n_bad_blocks;   /* blocks with a non-finite logit (nothing staged) */
  int64_t n_prev_transferred;  /* experts each routed layer transferred at its previous
                                  iteration (the effective transfer ratio's denominator) */
  int64_t n_transfers_reused;  /* of those, retained and activated again (its numerator,
                                  Sec. 5.3) */
  int64_t n_ideal_hits;   /* sum of min(C_l, |A|): hits of the clairvoyant ideal cache
                             bound (Sec. 5.1) */
  int64_t n_cpu_executed; /* misses executed on the CPU (apply_misses_coop) */
  int64_t n_miss_rows;    /* routed tokens of the misses (sum over misses of their routes) */
} oled_stats;

/*
 * Inspection of a layer (synchronises the device). Every pointer is a
 * caller-owned host array or NULL (skipped). The routing arrays describe the
 * most recent route_block call of the context; they are filled only if that
 * call was for `layer` (then `tokens` = its T, else 0).
 */
typedef struct {
  int32_t* topk_idx;          /* [T*k] expert of route r = t*k + j, slot order (logit desc, id asc) */
  float* gates;               /* [T*k] gate of route r (fp32) */
  int32_t* counts;            /* [E] routes per expert */
  int32_t* offsets;           /* [E+1] exclusive prefix sum of counts */
  int32_t* perm;              /* [T*k] sorted position -> route */
  int32_t* inv_perm;          /* [T*k] route -> sorted position */
  uint64_t* score_q;          /* [E] priority numerators of the last score_and_retain of `layer` */
  uint8_t* resident_before;   /* [E] R of the layer before its last execution */
  uint8_t* resident_after;    /* [E] committed R of the layer now */
  int32_t* slot_of;           /* [E] committed cache slot per expert, -1 if absent */
  int32_t tokens;
  int32_t n_active, n_hits, n_misses;
  int32_t capacity;           /* the layer's cache capacity now (min(C, E) unless adaptive) */
  int32_t reserved;
  uint64_t* retain_key;       /* [E] key of the last retention of `layer` (score_q under
                                 OLED_POLICY_PRIORITY; last activation / routes under LRU / LFU) */
  int32_t prev_transferred;   /* the last routing of `layer`: experts it transferred at its
                                 previous iteration, */
  int32_t reused_transfers;   /* and those of them retained and activated now */
  float* logits;              /* [T*E] fp32 logits of the gate GEMM, filled if the last routing
                                 of `layer` was route_block_gate (else untouched) */
  uint8_t* retained;          /* [E] the set the last score_and_retain of `layer` kept
                                 (Top_C of the retention rule, Sec. 4.2), before any eviction
                                 by a layer-adaptive re-sizing that followed it (Sec. 4.3);
                                 equals resident_after unless such a re-sizing shrank the layer */
} oled_layer_state;

/* One timed operation (see oled_config.profile_ops). */
typedef struct {
  int32_t kind;      /* oled_op_kind */
  int32_t layer;
  float ms;          /* device time between the events around the operation */
  int64_t bytes;     /* algorithmic device-memory bytes of the operation's compute */
  int64_t flops;     /* algorithmic flops */
  int64_t h2d_bytes; /* bytes it transferred host->device (shader transfer inside a
                        GEMM launch, a transfer-only launch, or copy-engine copies) */
} oled_op_time;

typedef enum {
  OLED_OP_ROUTE_TOPK = 0,
  OLED_OP_PERMUTE = 1,
  OLED_OP_FFN_UP = 2,        /* grouped gate/up GEMM + SiLU*up epilogue */
  OLED_OP_FFN_DOWN = 3,      /* grouped down GEMM */
  OLED_OP_COMBINE = 4,       /* combine + priority/retention launch after a forward */
  OLED_OP_SCORE_RETAIN = 5,
  OLED_OP_H2D = 6,           /* copy-engine copies of one apply_misses, or a
                                transfer-only launch */
  OLED_OP_FFN_DENSE_UP = 7,  /* dense-tile gate/up GEMM (bf16 experts with 65+ routed rows) */
  OLED_OP_FFN_DENSE_DOWN = 8, /* dense-tile down GEMM */
  OLED_OP_LAYER_ADAPT = 9,    /* layer-adaptive re-sizing of the capacities */
  OLED_OP_ROUTE_GEMM = 10     /* the gate GEMM of route_block_gate */
} oled_op_kind;

/* Creates a context: allocates the slot pool (L*min(C,E) + min(E, Tmax*k)
 * expert slots), the device cache state, routing scratch, pinned records, a
 * copy stream and events on cfg->device. The cache starts empty (R = {} for
 * every layer) with capacity min(C, E) per layer.
 * Errors: INVALID_ARG (bad field, host pool not pinned, adapt_period < 0),
 * UNSUPPORTED (shape, or adapt_period > 0 with n_layers > 1024),
 * OUT_OF_MEMORY, HIP. On error *ctx_out is NULL. */
oled_status oled_create(const oled_config* cfg, void** ctx_out);

/* Waits for outstanding work and frees everything the context owns. NULL ok. */
void oled_destroy(void* ctx);

/* Text of the last error of ctx (never NULL; empty if none). With ctx NULL,
 * the last failure of a call without a context (oled_create,
 * oled_route_noalloc) on the calling thread. */
const char* oled_last_error(const void* ctx);

/* Empties every layer's cache (R := {}) and restores capacity min(C, E), the
 * smoothed statistics and the iteration count, as at creation. Synchronises. Also
 * the way out after an OLED_ERR_HIP that left the device state unknown (a
 * failed launch, a wait past its deadline), which leaves the context refusing
 * route_block (OLED_ERR_STATE) until it is reset. */
oled_status oled_reset_cache(void* ctx);

/*
 * Failure injection, for tests of the host's error paths (no device work
 * fails; every kernel runs normally). Resets the enqueue count.
 *  copy_fail_at > 0: the copy_fail_at-th miss copy that apply_misses enqueues
 *  from now on (OLED_COPY_SDMA) is not enqueued and fails as a failed
 *  hipMemcpyAsync would, once; 0: off.
 *  wait_deadline_ms > 0: how long the host waits for miss copies and for
 *  route_block's published result before it gives up with OLED_ERR_HIP;
 *  0: the default, 60000 ms.
 *  Errors: INVALID_ARG (NULL ctx, a negative value).
 */
oled_status oled_set_fault_injection(void* ctx, int32_t copy_fail_at, int32_t wait_deadline_ms);

/*
 * route_block: the gate of Sec. 4.1 for the T tokens of the block.
 *  logits_dev: float [T][E] router logits. For each token the k largest
 *  logits are selected, ordered by (logit desc, expert id asc) (-0.0 equals
 *  +0.0); gate[t][j] = e_j / sum_j' e_j' with e_j = exp(l_j - l_0) in fp64,
 *  summed in slot order, rounded once to fp32. Then the expert histogram,
 *  exclusive offsets and the stable counting-sort permutation of the T*k
 *  routes by (expert, token). Asynchronous on `stream`.
 *  The same kernel splits the active experts into hits and misses against
 *  the layer's resident set and gives every miss a free staging slot.
 *  Errors: INVALID_ARG (layer outside [0,L), T outside [1,Tmax], NULL logits),
 *  STATE. A non-finite logit is detected on the device: nothing is staged and
 *  the layer's retention commits nothing; it is reported by apply_misses when
 *  a report is asked for, else by the next oled_read_layer_state of the layer
 *  (and counted by oled_collect_stats).
 */
oled_status route_block(void* ctx, int32_t layer, const float* logits_dev, int32_t T,
                        void* stream);

/*
 * route_block_gate: route_block with the gate in front (Sec. 2.1, 4.1: the
 *  MoE gate scores every token against every expert). x_dev: [T][H] dtype,
 *  the layer's input; w_gate_dev: [E][H] dtype, the gate weights (row e
 *  scores expert e). logits[t][e] = sum_h x[t][h] * w_gate[e][h], products
 *  exact, accumulated in fp32 in an order fixed by (T, E, H): each tile of
 *  tokens x experts splits the hidden dimension over its wavefronts and sums
 *  their partial tiles in wavefront order, so repeated calls give identical
 *  logits. They go to the context's logits buffer, then everything
 *  route_block does runs on them; oled_read_layer_state returns them.
 *  Errors: as route_block (NULL x or w_gate: INVALID_ARG).
 */
oled_status route_block_gate(void* ctx, int32_t layer, const void* x_dev, const void* w_gate_dev,
                             int32_t T, void* stream);

/*
 * moe_forward_cached: the cached experts of the routed layer (Sec. 4.1).
 *  x_dev: [T][H] dtype (read); y_dev: [T][H] dtype, written by the combine
 *  that score_and_retain enqueues: y[t] = sum_j gate[t][j] *
 *  W2_e (silu(W1_e x[t]) * (W3_e x[t])), e = idx[t][j] (lossless, Sec. 5.1).
 *  Enqueues the grouped GEMMs of the hit experts (A & R, weights read from
 *  their cache slots) on `stream` right away; their work list and count come
 *  from route_block's kernels on the device, so no host synchronisation is
 *  needed. With OLED_COPY_SHADER only their gate/up GEMM is enqueued here,
 *  and its first workgroups transfer the staged misses' gate/up weights; the
 *  hits' down GEMM follows in apply_misses. Accumulation is fp32;
 *  silu(W1 x) * (W3 x) is stored in dtype.
 *  Both buffers must stay valid until the layer's work has run.
 *  Errors: STATE (not right after route_block), INVALID_ARG (NULL pointers,
 *  a stream other than route_block's).
 */
oled_status moe_forward_cached(void* ctx, int32_t layer, const void* x_dev, void* y_dev,
                               void* stream);

/*
 * apply_misses: misses M = A \ R of the routed layer (Sec. 4.2) and their
 *  compensation by transfer (G = M), then the combine.
 *  OLED_COPY_SHADER: if moe_forward_cached was called, enqueues one launch
 *  holding the hits' down GEMM, the transfer of the misses' down weights and
 *  the misses' gate/up GEMM (their gate/up weights landed with the hits'
 *  gate/up launch), then the misses' down GEMM; else a transfer-only launch.
 *  Nothing waits for the device unless out is non-NULL. copy_stream is not
 *  used.
 *  OLED_COPY_SDMA: waits for route_block's result, copies every staged miss
 *  with hipMemcpyAsync on copy_stream (NULL: the context's own copy stream),
 *  gate/up weights of all misses first, then their down weights; if
 *  moe_forward_cached was called, launches the misses' GEMMs on the compute
 *  stream as the host sees each half of the copies land (the call returns
 *  once the last copy has landed).
 *  out (may be NULL): filled from the layer's routing record, which makes the
 *  call wait for route_block's kernel.
 *  Errors: STATE; INVALID_ARG if the record shows a non-finite logit (only
 *  seen when the record is read: with a report, or always with
 *  OLED_COPY_SDMA): nothing was staged, y is not written, the layer returns
 *  to idle with its cache unchanged. HIP if a miss copy could not be
 *  enqueued: the copies already enqueued are waited for, the staged misses
 *  return their slots, the layer's resident set, slot table and last
 *  retention keys stay as they were, y is not written and the layer returns
 *  to idle (the context stays usable). HIP if a launch failed, or a copy or
 *  the routing result did not complete within the wait deadline (60 s by
 *  default): the device state is then unknown and the context needs
 *  oled_reset_cache. Retentions enqueued earlier that were rejected for an
 *  invalid confidence are named in out->rejected_layer (the call still
 *  returns OLED_OK for its own work).
 */
oled_status apply_misses(void* ctx, int32_t layer, void* copy_stream, oled_miss_report* out);

/*
 * score_and_retain: priorities of Sec. 4.3 and the retention rule of Sec. 4.2.
 *  (With oled_config.policy LRU or LFU the candidates are ranked by that key
 *  instead of S; S is still computed and reported.)
 *  conf_dev: float [T] token confidence in [0, 1]. For each expert,
 *  S[e] = sum over its routes of floor(fp64(gate) * fp64(conf[t]) * 2^48)
 *  (exact; p_e = S[e] / sum S). Residents that no token routed to score 0.
 *  Candidates R u M are ranked by (S desc, previously resident first, id asc)
 *  and the first min(C, |R u M|) stay cached for the next iteration of this
 *  layer; the rest release their slots. The same kernel commits the new
 *  state in device memory (retained misses keep their staging slot). After
 *  moe_forward_cached its launch also holds the combine into y.
 *  Errors: STATE, INVALID_ARG (NULL conf). A confidence outside [0,1] (or NaN)
 *  is detected on the device: the layer keeps its previous R, its transferred
 *  misses are dropped, and the rejection is reported by the next report of
 *  apply_misses (rejected_layer) and by oled_read_layer_state.
 *
 *  Layer-adaptive sizing (oled_config.adapt_period > 0; Sec. 4.3, the layer
 *  weight w_l = a_l * u_l and the capacity C_l = C_total * w_l / sum_j w_j).
 *  C is then the layer's current capacity C_l. Each committed retention also
 *  folds the layer's routing into its smoothed statistics (float64,
 *  x <- obs/2 + x/2 from the first observation): activation ratio |A| / E and
 *  utilisation hits / C_l (skipped while C_l = 0). After the retention of
 *  layer L-1 that completes every adapt_period-th iteration (counted from
 *  creation or oled_reset_cache), the same stream gets one more launch that
 *  re-sizes all layers: proportional shares of C_total, none above E (the
 *  excess re-shared), rounded by the largest remainder (ties to the lower
 *  layer); if every w_l is 0 nothing changes. A layer now holding more than
 *  its new C_l evicts its residents of lowest priority at once (its last
 *  numerators S desc, id asc), so the layers never hold more than C_total
 *  experts; a layer that grew fills its room at its next retentions.
 */
oled_status score_and_retain(void* ctx, int32_t layer, const float* conf_dev, void* stream);

/*
 * apply_misses_coop: cooperative compensation of the routed layer's misses
 *  (Sec. 4.4), in place of apply_misses on a context created with coop = 1.
 *  On such a context moe_forward_cached launches the hits' gate/up GEMM
 *  without copying any miss, and copies x to pinned host memory on the
 *  context's copy stream; the routing kernel publishes the layer's routes
 *  with its staged misses. apply_misses_coop waits for them; if there are
 *  misses it copies conf_dev (float [T], the same confidence
 *  score_and_retain gets) to the host and computes:
 *   - priorities S_e as in score_and_retain (exact integers);
 *   - the hardware-aware split rho = nbar tau / (nbar tau + T_H2D) and the
 *     two-stage dispatch of oled_coop_dispatch: the transfer set G;
 *   - the staging slots of the CPU experts M minus G return to the free list
 *     (one launch); the hits' down GEMM copies G's whole blocks in its first
 *     workgroups, then G's GEMMs run on the GPU;
 *   - the CPU experts run on coop_threads host threads from the pinned pool
 *     (oled_cpu_ffn's kernels); their output rows are copied into the
 *     layer's per-route outputs before the combine (stream order). The call
 *     returns once those copies are enqueued.
 *  score_and_retain then keeps Top_C of R u G: CPU-executed experts never
 *  enter the cache. out (may be NULL) reports the layer's counts; its
 *  h2d_bytes are G's.
 *  Errors: STATE (not in flight, or not a coop context), INVALID_ARG (NULL
 *  conf, or a bad block as in apply_misses), HIP.
 */
oled_status apply_misses_coop(void* ctx, int32_t layer, const float* conf_dev,
                              oled_miss_report* out);

/*
 * oled_coop_dispatch: the dispatch of Sec. 4.4 on host arrays (the same code
 *  apply_misses_coop runs). miss [E] (nonzero: a miss), n_tok [E] routed
 *  tokens, score [E] priority numerators of every expert of the layer.
 *  rho = nbar tau / (nbar tau + T_H2D) (1 if that is 0/0); stage 1 marks the
 *  round_half_up(rho |M|) misses of highest (score desc, id asc); stage 2
 *  makes at most |M| swaps of a transferred and a CPU expert, each the best
 *  by J(G) = max(T_H2D |G|, tau * CPU tokens) - lambda * (sum_G S / sum S)
 *  (first in (transferred id, CPU id) order among equals) and only if it
 *  lowers J. float64, in that order of operations. transfer_out [E]: 1 for G.
 *  Errors: INVALID_ARG (NULL pointers, E outside [1, 256], negative times).
 */
oled_status oled_coop_dispatch(int32_t n_experts, const uint8_t* miss, const int32_t* n_tok,
                               const uint64_t* score, double t_h2d_us, double tau_cpu_us,
                               double nbar, double lambda_us, uint8_t* transfer_out);

/*
 * oled_cpu_ffn: one expert's SwiGLU on the host CPU (the kernels of the
 *  cooperative compensation). block: packed expert block (oled_pack_expert
 *  layout, dtype); x: [n][H] token rows in dtype; out: [n][H] fp32.
 *  Accumulates in fp32; silu(W1 x) * (W3 x) is rounded to dtype as the GPU
 *  stores it. threads >= 1 host threads: the first call with a given count
 *  starts them, later calls reuse them (calls from several threads take
 *  turns). Needs AVX2 and FMA; bf16 uses AVX-512 BF16 dot products where the
 *  CPU has them (environment OLED_CPU_FFN_AVX2=1 forces the AVX2 kernels).
 *  Errors: INVALID_ARG (NULL pointers, n < 0, threads < 1, bad dtype),
 *  UNSUPPORTED (shape, or the CPU lacks AVX2/FMA).
 */
oled_status oled_cpu_ffn(int32_t dtype, int32_t hidden, int32_t inter, const void* block,
                         const void* x, int32_t n, float* out, int32_t threads);

/* Inspection (synchronises; see oled_layer_state). With no layer in flight it
 * also checks slot conservation over the whole device cache state (every
 * slot free or held by exactly one resident expert, |R| <= C_l per layer,
 * capacities within [0, E] summing to at most C_total) and
 * returns HIP if it does not hold. Returns INVALID_ARG (with the arrays
 * filled) if the layer's last retention was rejected, or once after a bad
 * block of the layer that no report has named. */
oled_status oled_read_layer_state(void* ctx, int32_t layer, oled_layer_state* out);

/* Totals of the routing records since the last call (synchronises). */
oled_status oled_collect_stats(void* ctx, oled_stats* out);

/* Operation timings recorded since the last collection (oled_config.profile_ops).
 * Synchronises. Writes at most cap entries to out, sets *n_out; entries that
 * did not fit are dropped. */
oled_status oled_profile_collect(void* ctx, oled_op_time* out, int32_t cap, int32_t* n_out);

/*
 * Packs one expert's logical weights into an expert block of the host pool.
 *  w13: [2I][H] row-major (gate projection W1 rows 0..I-1, then up projection
 *  W3 rows); w2: [H][I] row-major; elements of `dtype` (bf16 as raw 16-bit
 *  patterns). block_out: 3*H*I elements, written in the order the grouped
 *  GEMM reads them. With SPAN = 32 (bf16) or 16 (fp32), V = SPAN/4, S = H/SPAN
 *  and S2 = I/SPAN, a fragment holds 16 rows x SPAN columns as element
 *  l*V + i <- (row 16q + l%16, column SPAN*s + V*(l/16) + i), l < 64, i < V:
 *    gate/up part: fragment ((q*S + s)*2 + m), m = 0 for W1, 1 for W3, q < I/16;
 *    down part, after 2*I*H elements: fragment (q*S2 + s) of w2, q < H/16.
 *  Host only; never fails for valid shapes (H, I multiples of 128).
 *  Errors: INVALID_ARG (NULL pointer, bad dtype), UNSUPPORTED (shape).
 */
oled_status oled_pack_expert(int32_t dtype, int32_t hidden, int32_t inter, const void* w13,
                             const void* w2, void* block_out);

/*
 * Routing and permutation of one block without a context and without any
 * allocation: for callers that cannot allocate device memory (code under HIP
 * graph capture, serving loops and harnesses that forbid hipMalloc). It
 * computes what route_block computes before the cache is consulted, with the
 * same kernels and bit-identical results: top-k ids and fp64-evaluated gates
 * (one fp32 rounding, slot order logit desc / id asc), the expert histogram,
 * exclusive offsets and the stable permutation. There is no expert cache:
 * no hit/miss split, staging or records.
 *  logits_dev [T][E] fp32 (read); topk_idx_dev [T*k] int32, gates_dev [T*k]
 *  fp32, counts_dev [E], offsets_dev [E+1], perm_dev [T*k] (sorted position ->
 *  route), inv_perm_dev [T*k] (route -> position), all int32 except gates,
 *  caller-owned device memory on the current device, overwritten.
 *  nonfinite_dev: optional int32 written 1 if a logit was NaN or infinite
 *  (the other outputs are then unspecified), else 0.
 *  stream: a stream of the current device (NULL: the null stream).
 * Limits: 1 <= T <= 65535, 1 <= k <= E <= 256, k <= 16 (UNSUPPORTED beyond
 * them, INVALID_ARG for a NULL output or T, E, k below 1; the text is in
 * oled_last_error(NULL)). The launches' counters and per-chunk counts live in
 * one file-scope device array of oled_route_noalloc_scratch_bytes() bytes
 * (about 128 KiB), one copy per GPU, held until the process ends; the call
 * clears what must start at zero with a small kernel (no memset node), so it
 * can be captured. Calls on one GPU share that array: calls whose work
 * overlaps on the device (concurrent streams, or threads) race; calls in
 * one stream's order do not. Returns HIP if a launch fails.
 */
oled_status oled_route_noalloc(const float* logits_dev, int32_t T, int32_t E, int32_t k,
                               int32_t* topk_idx_dev, float* gates_dev, int32_t* counts_dev,
                               int32_t* offsets_dev, int32_t* perm_dev, int32_t* inv_perm_dev,
                               int32_t* nonfinite_dev, void* stream);
size_t oled_route_noalloc_scratch_bytes(void);

/*
 * The gate's routing (Sec. 4.1) and the expert histogram, offsets and stable
 * permutation (the active set of Sec. 4.2) of B independent blocks of T
 * tokens in one pass, without a context or an expert cache: for work over
 * many blocks whose logits are all at hand (replaying recorded routing of
 * many layers or requests, as policy studies do, Sec. 5.3). Block b's results
 * are bit-identical to route_block on block b alone.
 *  logits_dev [B][T][E] fp32; outputs, per block b at offset b*T*k (routes),
 *  b*E (counts), b*(E+1) (offsets): topk_idx_dev [B][T*k] int32, gates_dev
 *  [B][T*k] fp32, counts_dev [B][E], offsets_dev [B][E+1], perm_dev [B][T*k]
 *  (position within the block -> route within the block), inv_perm_dev
 *  [B][T*k]; nonfinite_dev: optional int32 [B], 1 where a block has a NaN or
 *  infinite logit (its other outputs are then unspecified), else 0. All
 *  caller-owned device memory, overwritten.
 *  workspace_dev: caller-owned device memory of at least
 *  oled_route_batch_workspace(B, T, E) bytes (counters and per-chunk counts;
 *  the call clears what must start at zero); nothing is allocated.
 * Limits: 1 <= T <= 65535, 1 <= k <= E <= 256, k <= 16, B*T*k < 2^31
 * (UNSUPPORTED beyond them; INVALID_ARG for NULL pointers, sizes below 1 or a
 * short workspace, with the text in oled_last_error(NULL)). Calls that share
 * a workspace must not overlap on the device.
 */
oled_status oled_route_batch(const float* logits_dev, int32_t B, int32_t T, int32_t E, int32_t k,
                             int32_t* topk_idx_dev, float* gates_dev, int32_t* counts_dev,
                             int32_t* offsets_dev, int32_t* perm_dev, int32_t* inv_perm_dev,
                             int32_t* nonfinite_dev, void* workspace_dev, size_t workspace_bytes,
                             void* stream);
size_t oled_route_batch_workspace(int32_t B, int32_t T, int32_t E);

/*
 * The reuse-priority numerators of the priority equation of Sec. 4.3
 * (psi(c) = c) of B independent blocks in one pass, without retention:
 * score_q[b][e] = sum over routes r of block b with topk_idx[b][r] = e of
 * floor(gate[b][r] * conf[b][r / k] * 2^48), exact in uint64 (the values
 * score_and_retain computes for one block).
 *  topk_idx_dev, gates_dev [B][T*k] as oled_route_batch writes them; conf_dev
 *  [B][T] fp32 in [0, 1]; score_q_dev [B][E] uint64, overwritten;
 *  bad_conf_dev: optional int32 [B], 1 where a block has a confidence outside
 *  [0, 1] (its numerators are then unspecified), else 0.
 * Limits and errors as oled_route_batch (T <= 65535 keeps every sum below
 * 2^64). Nothing is allocated.
 */
oled_status oled_priority_batch(const int32_t* topk_idx_dev, const float* gates_dev,
                                const float* conf_dev, int32_t B, int32_t T, int32_t E, int32_t k,
                                uint64_t* score_q_dev, int32_t* bad_conf_dev, void* stream);

/* Pinned host memory for expert pools (hipHostMalloc). *ptr_out NULL on error. */
oled_status oled_host_alloc(int64_t bytes, void** ptr_out);
void oled_host_free(void* ptr);

#ifdef __cplusplus
}
#endif

#endif /* OLED_H_ */
