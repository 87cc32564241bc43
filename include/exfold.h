/*
 * exfold.h -- C-ABI of libexfold, the ExFold folded mixture-of-experts layer
 * for AMD Instinct MI355X (gfx950).
 *
 * Method: arXiv 2608.24938, "ExFold: Unified Expert Folding for Training-Free
 * MoE Prefill-Decode Acceleration".  The layer routes each token to its Top-K
 * experts (Sec. 2.1, Eq. topk_gate), keeps a phase-specific retained set
 * (Sec. 4.3 step 1: per token in prefill, Eq. prefill_budget; per batch in
 * decode, Eq. decode_budget), folds every omitted route onto its minimum-loss
 * retained target through a calibrated scalar (Sec. 4.3 steps 2-3,
 * Eq. minimum_loss_assignment, Eq. prefill_fold, Eq. decode_remap), and runs
 * the SwiGLU experts (Eq. gated_expert) of the retained routes only, combining
 * them with the folded weights (Eq. moe_output, Eq. folded_moe).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.    Every tensor pointer is caller-owned DEVICE memory, contiguous and
 *            row-major, unless stated otherwise.  Outputs and workspaces are
 *            allocated by the caller; the library allocates no device memory
 *            and keeps no state besides a read-only cache of device properties
 *            and the static scratch of exfold_moe_forward_scratch.
 *            The layer's weights and the token tensors x, y and x_cal are read
 *            and written in 16-byte vectors: their base pointers must be
 *            16-byte aligned (else EXFOLD_ERR_ALIGN).
 * Streams.   `stream` is a hipStream_t passed as void* (NULL: the null stream).
 *            Every call only enqueues work and returns: no host synchronisation
 *            and no device-to-host copy.
 * Errors.    All arguments are validated on the host BEFORE anything is
 *            enqueued, so a call that returns an error has written nothing.
 *            EXFOLD_ERR_DEVICE reports a failed kernel launch.  Data never
 *            causes an error: any finite input is valid; non-finite inputs give
 *            unspecified values, but every expert id a kernel reads is clamped
 *            to [0, N), so no input can cause an out-of-bounds access.
 * Limits.    1 <= K <= 16, K <= N <= 256, d % 128 == 0, I % 64 == 0 (else
 *            EXFOLD_ERR_UNSUPPORTED); the shared expert, if present, must have
 *            I_s == I (else EXFOLD_ERR_UNSUPPORTED).  T == 0 is a valid no-op; T <= 2^22.
 * Budgets.   K' < 1 or D < 1 is EXFOLD_ERR_BUDGET.  K' >= K, or D >= the number
 *            of distinct routed experts, leaves the routes unchanged bit for bit.
 * Order.     Top-K routes are ordered by (logit descending, expert id ascending).
 *            Identical inputs give bit-identical outputs on the same device.
 * Dtypes.    EXFOLD_BF16: x, y and all weights are bf16 (raw 16-bit storage);
 *            EXFOLD_F32: all float32.  Router logits, gate weights, the S, L and
 *            h tables and router bias are always float32.
 */
#ifndef EXFOLD_H
#define EXFOLD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t exfold_status;

enum {
  EXFOLD_OK = 0,
  EXFOLD_ERR_NULL = 1,         /* a required pointer is NULL                      */
  EXFOLD_ERR_SHAPE = 2,        /* a size is negative, inconsistent or too large   */
  EXFOLD_ERR_BUDGET = 3,       /* K' < 1 or D < 1                                 */
  EXFOLD_ERR_DTYPE = 4,        /* unknown dtype code                              */
  EXFOLD_ERR_WORKSPACE = 5,    /* workspace smaller than required or misaligned   */
  EXFOLD_ERR_DEVICE = 6,       /* a HIP launch or query failed                    */
  EXFOLD_ERR_UNSUPPORTED = 7,  /* valid request outside the kernels' limits       */
  EXFOLD_ERR_ARG = 8,          /* unknown phase or mode, or invalid scalar arg    */
  EXFOLD_ERR_ALIGN = 9,        /* a tensor pointer is not 16-byte aligned         */
  EXFOLD_ERR_SCRATCH = 10      /* needs more than EXFOLD_SCRATCH_BYTES of scratch */
};

enum { EXFOLD_F32 = 0, EXFOLD_BF16 = 1 };

enum {
  EXFOLD_PHASE_DENSE = 0,    /* unfolded layer on the Top-K routes (Eq. moe_output)  */
  EXFOLD_PHASE_PREFILL = 1,  /* per-token K' budget (Eq. prefill_budget/prefill_fold) */
  EXFOLD_PHASE_DECODE = 2,   /* per-batch pool of D (Eq. decode_budget/decode_remap)  */
  EXFOLD_PHASE_DECODE_STATIC = 3, /* static pool of D: remap with precomputed tables
                                     (Appendix B, Eq. appendix_decode_static_budget,
                                     Eq. appendix_decode_remap); see exfold_static_pool */
  EXFOLD_PHASE_PREFILL_DIAG = 4   /* per-token K' budget with diagonal projectors on the
                                     unfused path (Appendix B,
                                     Eq. appendix_diagonal_projector); see
                                     exfold_calibrate_diagonal */
};

enum {
  EXFOLD_CAL_COROUTED = 0,  /* outputs of co-routed experts only (Sec. 4.2)            */
  EXFOLD_CAL_COMMON = 1     /* every expert on every calibration token (common input) */
};

/* Prefill fold safeguards (bits of exfold_tables.fold_flags and of the
 * fold_flags argument of exfold_fold_gates); 0 = the main method.
 *   LOSS_CAP:   a pair (s, t) with L[s, t] > loss_cap is not a candidate target;
 *               an omitted route with no candidate is dropped (Appendix C:
 *               directed pairs with calibrated loss above 0.99 excluded).
 *   RENORM:     after folding, the retained weights are scaled by (sum of the K
 *               router weights) / (sum of the folded weights) when that sum is
 *               positive (Appendix C: the routed-weight sum is preserved).
 *   CONFIDENCE: c_s = clip(1 - min_t L[s, t], 0, 1); the target receives
 *               w_s c_s S[s, t] and w_s (1 - c_s) is spread over the retained
 *               routes in proportion to their router weights (Appendix F,
 *               Eq. dsv4_confidence, with L as the source-relative residual).
 * Safeguard arithmetic is float64, rounded once to float32 (see the oracle's
 * fold_prefill_safeguarded for the order of operations). */
enum { EXFOLD_FOLD_LOSS_CAP = 1, EXFOLD_FOLD_RENORM = 2, EXFOLD_FOLD_CONFIDENCE = 4 };

/* One MoE layer.  Pointers are device memory of dtype `dtype` unless noted. */
typedef struct exfold_layer {
  int64_t d;              /* hidden size                                          */
  int64_t inter;          /* expert intermediate size I                           */
  int64_t n_experts;      /* routed experts N                                     */
  int64_t top_k;          /* router Top-K                                         */
  int64_t shared_inter;   /* shared-expert intermediate size I_s; 0 = no shared   */
  int32_t dtype;          /* EXFOLD_BF16 or EXFOLD_F32                            */
  int32_t reserved;
  const void *w_router;     /* [N, d]                                               */
  const float *router_bias; /* [N] float32 added to the logits, or NULL             */
  const void *w_gate_up;    /* [N, 2I, d]: rows 0..I-1 W_gate, rows I..2I-1 W_up   */
  const void *w_down;       /* [N, d, I]                                            */
  const void *ws_gate_up;   /* [2I_s, d] shared expert, or NULL                     */
  const void *ws_down;      /* [d, I_s] shared expert, or NULL                      */
} exfold_layer;

/* Calibrated per-layer tables (Sec. 4.2): S[s*N+t] = s*_{s->t}, L[s*N+t] = l_{s->t}
 * (row = source s, column = target t), h[e] = output-norm estimate of expert e.
 * tgt/scl: the per-source tables of a static decode pool (exfold_static_pool);
 * required by EXFOLD_PHASE_DECODE_STATIC, ignored (may be NULL) otherwise. */
typedef struct exfold_tables {
  const float *S;      /* [N, N] float32 */
  const float *L;      /* [N, N] float32 */
  const float *h;      /* [N]    float32 */
  const int32_t *tgt;  /* [N]    int32: target of each source expert, or NULL */
  const float *scl;    /* [N]    float32: its scale, or NULL                  */
  float loss_cap;      /* prefill: cap of EXFOLD_FOLD_LOSS_CAP                */
  int32_t fold_flags;  /* prefill: EXFOLD_FOLD_* safeguards, 0 = none         */
  const float *Dg;     /* [N, N, d] diagonal maps d_{s->t} (Dg[(s*N+t)*d+n]) for
                          EXFOLD_PHASE_PREFILL_DIAG, whose L is then the diagonal
                          loss table; NULL otherwise                          */
} exfold_tables;

/* Stage boundaries at which exfold_moe_forward records the optional events. */
enum {
  EXFOLD_EV_START = 0,    /* before the router                                  */
  EXFOLD_EV_ROUTER = 1,   /* after the router logits                            */
  EXFOLD_EV_FOLD = 2,     /* after Top-K, selection and folding                 */
  EXFOLD_EV_PERMUTE = 3,  /* after the permutation                              */
  EXFOLD_EV_GATE_UP = 4,  /* after the gate/up GEMM with fused SiLU * up        */
  EXFOLD_EV_DOWN = 5,     /* after the down GEMM                                */
  EXFOLD_EV_END = 6,      /* after the combine (== EXFOLD_EV_DOWN when fused)   */
  EXFOLD_N_EVENTS = 7
};

/* Optional views of the forward's intermediates.  A non-NULL pointer is used
 * as the buffer of that intermediate (no extra copy); NULL members live in the
 * workspace.  Sizes: K_out = min(K', K) in prefill, K otherwise.
 * `events`, if non-NULL, holds EXFOLD_N_EVENTS hipEvent_t handles (created by
 * the caller) that are recorded on the stream at the stage boundaries above;
 * a NULL entry is skipped (no event at that boundary). */
typedef struct exfold_debug {
  float *logits;        /* [T, N]      router logits                                   */
  int32_t *topk_ids;    /* [T, K]      Top-K expert ids                                */
  float *topk_w;        /* [T, K]      renormalised gate weights                       */
  uint8_t *keep;        /* [T, K]      prefill: 1 = retained route                     */
  int32_t *pool;        /* [min(D,N)]  decode pool, -1 padded                           */
  int32_t *pool_size;   /* [1]         decode pool size                                 */
  int32_t *tgt_ids;     /* [N]         decode target of each source expert              */
  float *tgt_scale;     /* [N]         decode scale of each source expert               */
  int32_t *fold_ids;    /* [T, K_out]  folded route ids                                 */
  float *fold_w;        /* [T, K_out]  folded route weights                             */
  int32_t *offsets;     /* [N+2]       row offsets of each expert group (+ shared rows) */
  int32_t *row_slot;    /* [R]         flat route slot i*K_out+k executed by each row   */
  void *const *events;  /* [EXFOLD_N_EVENTS] hipEvent_t, or NULL                        */
} exfold_debug;

/*
 * Prefill selection (Eq. topk_gate, Eq. prefill_budget).
 *   logits   [T, N] float32, or NULL: then topk_ids/topk_w are INPUTS.
 *   topk_ids [T, K] int32, topk_w [T, K] float32: outputs when logits != NULL
 *            (Top-K by (logit desc, id asc); softmax over the K selected logits,
 *            evaluated in float64 and rounded once to float32).
 *   h        [N] float32 output-norm estimates.
 *   keep     [T, K] uint8 output: 1 for the K' routes of largest w*h (the exact
 *            float64 product; equal scores keep the smaller route position).
 */
exfold_status exfold_select_prefill(const float *logits, int64_t T, int64_t N, int64_t K,
                                    int64_t k_pre, const float *h, int32_t *topk_ids,
                                    float *topk_w, uint8_t *keep, void *stream);

/*
 * Decode pool selection (Eq. topk_gate, Eq. decode_budget).
 *   logits    [B, N] float32, or NULL: then topk_ids/topk_w are INPUTS [B, K].
 *   pool      [min(D, N)] int32 output: the retained pool in (score desc, id asc)
 *             order, -1 padded.  Candidates are the experts with >= 1 routed
 *             slot; score_e = fl64(W_e * h_e) with W_e = sum of rint(w * 2^40)
 *             over the slots routed to e (an exact integer).
 *   pool_size [1] int32 output: min(D, number of candidates).
 */
exfold_status exfold_select_decode_pool(const float *logits, int64_t B, int64_t N, int64_t K,
                                        int64_t D, const float *h, int32_t *topk_ids,
                                        float *topk_w, int32_t *pool, int32_t *pool_size,
                                        void *stream);

/*
 * Fold router metadata (Eq. minimum_loss_assignment with Eq. prefill_fold or
 * Eq. decode_remap).  The target of an omitted source s is the first minimum of
 * L[s, t] over the retained set in canonical order (route order in prefill,
 * pool order in decode).
 *   PREFILL: keep [T, K] from exfold_select_prefill; budget = K'.  Outputs
 *            out_ids/out_w [T, min(K', K)]: retained routes in route order with
 *            w~_t = w_t + sum of w_s * S[s, t] over the omitted s folded onto t
 *            (omitted routes visited in route order, float64 sum rounded once).
 *   DECODE:  pool/pool_size from exfold_select_decode_pool; budget = D.
 *            Outputs out_ids/out_w [T, K], layout unchanged: a slot of source s
 *            outside the pool becomes (tgt[s], w * S[s, tgt[s]]) with one float32
 *            multiply; retained slots are copied.  tgt_ids/tgt_scale [N] are
 *            optional outputs of the per-source tables (NULL to skip).
 *   loss_cap/fold_flags: PREFILL safeguards (EXFOLD_FOLD_*); ignored in DECODE.
 *   Unused arguments of the other phase may be NULL.
 */
exfold_status exfold_fold_gates(int32_t phase, int64_t T, int64_t N, int64_t K, int64_t budget,
                                const int32_t *topk_ids, const float *topk_w,
                                const uint8_t *keep, const int32_t *pool,
                                const int32_t *pool_size, const float *S, const float *L,
                                int32_t *out_ids, float *out_w, int32_t *tgt_ids,
                                float *tgt_scale, float loss_cap, int32_t fold_flags,
                                void *stream);

/*
 * Static decode pool (Appendix B, Eq. appendix_decode_static_budget): formed
 * once from the calibration norms, independent of the batch.
 *   h         [N] float32 output-norm estimates.
 *   pool      [min(D, N)] int32 output: the D experts of largest h in (h desc,
 *             id asc) order.  pool_size [1] int32 output: min(D, N).
 *   tgt, scl  [N] outputs: the per-source tables of this pool (a source in the
 *             pool maps to itself with scale 1; any other source s to the first
 *             minimum t of L[s, t] over the pool in pool order, with scale
 *             S[s, t]).  Pass them as exfold_tables.tgt/scl to an
 *             EXFOLD_PHASE_DECODE_STATIC forward, whose per-step fold is then
 *             one lookup per routed slot (Eq. appendix_decode_remap).
 */
exfold_status exfold_static_pool(const float *h, int64_t N, int64_t D, const float *S,
                                 const float *L, int32_t *pool, int32_t *pool_size, int32_t *tgt,
                                 float *scl, void *stream);

/* Bytes of workspace exfold_moe_forward needs for T tokens, or 0 on invalid input. */
size_t exfold_moe_workspace_size(const exfold_layer *layer, int64_t T, int32_t phase,
                                 int64_t budget);

/*
 * Folded MoE layer forward (Sec. 4.3 end to end): router logits, Top-K softmax,
 * phase selection, fold, stable permutation of the executed routes by expert,
 * grouped SwiGLU expert GEMMs over the retained routes only, weighted combine.
 *   x   [T, d] input tokens, y [T, d] output (same dtype as the layer).
 *   tables may be NULL for EXFOLD_PHASE_DENSE; budget is ignored there.
 *   EXFOLD_PHASE_PREFILL_DIAG needs tables->h, L (the diagonal loss) and Dg from
 *   exfold_calibrate_diagonal: the K' routes of largest w*h execute with their
 *   router weights w_t, each omitted route s goes to the first minimum of L[s, t]
 *   over them, and y_i = sum_t (w_t + sum of w_s Dg[s, t]) . E_t(x_i) (+ shared).
 *   EXFOLD_PHASE_DECODE_STATIC needs tables->tgt/scl from exfold_static_pool
 *   (budget = its D) and leaves the debug pool/pool_size/tgt_ids/tgt_scale
 *   untouched; a slot of source s becomes (tgt[s], w * scl[s]) unless tgt[s] == s.
 *   y_i = sum over executed routes (e, w) of w * E_e(x_i), plus the shared
 *   expert with weight 1; float32 accumulation, one rounding to the dtype.
 *   debug may be NULL.  ws/ws_bytes: workspace of at least
 *   exfold_moe_workspace_size bytes, 256-byte aligned.
 */
exfold_status exfold_moe_forward(const exfold_layer *layer, const exfold_tables *tables,
                                 const void *x, int64_t T, int32_t phase, int64_t budget,
                                 void *y, const exfold_debug *debug, void *ws, size_t ws_bytes,
                                 void *stream);

/*
 * exfold_moe_forward without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops and harnesses
 * that forbid hipMalloc).  The call allocates nothing: its intermediates live
 * in a static scratch array of EXFOLD_SCRATCH_BYTES inside the library, one
 * copy per GPU, held from the library's first use on that GPU until the
 * process ends.  Arguments, outputs and errors are those of
 * exfold_moe_forward (debug views included), plus EXFOLD_ERR_SCRATCH when
 * exfold_moe_workspace_size(layer, T, phase, budget) > EXFOLD_SCRATCH_BYTES
 * (returned before anything is enqueued).  Results are bit-identical to
 * exfold_moe_forward's.  Every call on one GPU uses that GPU's single array,
 * which keeps the last call's contents: calls that overlap on one GPU (other
 * streams or host threads) race and must be serialised by the caller.
 */
#define EXFOLD_SCRATCH_BYTES ((size_t)64 << 20)
exfold_status exfold_moe_forward_scratch(const exfold_layer *layer, const exfold_tables *tables,
                                         const void *x, int64_t T, int32_t phase, int64_t budget,
                                         void *y, const exfold_debug *debug, void *stream);

/* Bytes of workspace exfold_moe_execute needs for T tokens of K_out routes. */
size_t exfold_execute_workspace_size(const exfold_layer *layer, int64_t T, int64_t k_out);

/*
 * Execute given route metadata (the expert stage that the fold feeds, Eq.
 * moe_output on arbitrary routes): route_ids/route_w [T, K_out] (ids in [0, N),
 * duplicates allowed, any weights).  y as in exfold_moe_forward.  debug may be
 * NULL; only its offsets/row_slot members are used.
 */
exfold_status exfold_moe_execute(const exfold_layer *layer, const void *x, int64_t T,
                                 int64_t k_out, const int32_t *route_ids, const float *route_w,
                                 void *y, const exfold_debug *debug, void *ws, size_t ws_bytes,
                                 void *stream);

/* Bytes of workspace exfold_calibrate_projectors (and exfold_calibrate_diagonal)
 * needs for m calibration tokens. */
size_t exfold_calibrate_workspace_size(const exfold_layer *layer, int64_t m, int32_t mode);

/*
 * Projector calibration (Sec. 4.2, Eq. calibration_outputs, Eq. scalar_projector,
 * Eq. projection_loss; Appendix A protocol; Appendix B Eq. A1-A2).
 *   x_cal [m, d] calibration tokens.  COROUTED: u = E_s(x), v = E_t(x) for the
 *   ordered pairs s != t of each token's Top-K experts; COMMON: for all pairs.
 *   Per pair, with w = ||u||_2: A = sum w<u,v>, V = sum w||v||^2,
 *   C = sum w||u||^2, n = count (float64, token order).
 *   S[s,t] = A/(V+lambda) (0 if n == 0 or V+lambda == 0), clipped to
 *   [-clip, clip] when clip > 0; L[s,t] = max(0, C - 2 S A + S^2 V)/(C + 1e-12)
 *   with the clipped S, 1e30 when n == 0; S[s,s] = 1, L[s,s] = 0.
 *   h[e] = mean ||E_e(x)||_2 over the tokens on which E_e was evaluated; an
 *   expert never evaluated gets the mean of the observed h.
 *   Outputs S, L [N, N] and h [N] float32 (rounded once from float64);
 *   pair_stats [N, N, 4] float64 (A, V, C, n) optional (NULL to skip).
 *   lambda >= 0 and clip >= 0 are required (else EXFOLD_ERR_ARG).
 */
exfold_status exfold_calibrate_projectors(const exfold_layer *layer, const void *x_cal, int64_t m,
                                          double lambda, double clip, int32_t mode, float *S,
                                          float *L, float *h, double *pair_stats, void *ws,
                                          size_t ws_bytes, void *stream);

/* Static text for a status code. */
const char *exfold_status_str(exfold_status status);

/* Kernel families of the expert GEMMs (exfold_gemm_plan). */
enum {
  EXFOLD_GEMM_SIMT = 0,    /* float32 layers                                          */
  EXFOLD_GEMM_TILE = 1,    /* 128x128 MFMA tiles                                      */
  EXFOLD_GEMM_SKINNY = 2,  /* 32x64 tiles streaming weights (few rows per expert)     */
  EXFOLD_GEMM_WIDE = 3     /* 256x256 tiles (128x512 tails) in rounds of one per CU   */
};

/*
 * Host-only query of the expert-GEMM plan the library takes for `rows`
 * executed rows (routed slots plus shared-expert rows) of a layer, when about
 * `active_groups` expert groups are non-empty, on a device with `cu_count`
 * compute units (the forward uses the device's count).  No device call.
 * out[10] = { gate_up: kind, bm, bn, ksplit, grid,  down: kind, bm, bn, ksplit, grid }
 * (kind an EXFOLD_GEMM_* value; bm the tile height, or for EXFOLD_GEMM_WIDE the
 * 128-row unit of its tile list; bn the tile width in output columns, or
 * weight rows for gate/up; grid the workgroups launched, an upper bound on the
 * tiles any split of the rows into groups can produce, plus for
 * EXFOLD_GEMM_WIDE one round for the split remainder).  The forward drops the
 * down split (ksplit 1) when each token owns one row or the rows are kept.
 * Errors: the layer's validation codes; EXFOLD_ERR_NULL for out == NULL;
 * EXFOLD_ERR_SHAPE for rows < 0, active_groups < 1 or cu_count < 1.
 */
exfold_status exfold_gemm_plan(const exfold_layer *layer, int64_t rows, int64_t active_groups,
                               int32_t cu_count, int32_t *out);

/*
 * Diagonal projector calibration (Appendix B, Eq. appendix_diagonal_projector;
 * the unfused family of the projector ablation).  Routing, evaluated pairs and
 * the weight w = ||u||_2 are those of exfold_calibrate_projectors.  Per ordered
 * pair (s, t), in token order and float64, per hidden dimension n:
 *   A_n = sum w v_n u_n, V_n = sum w v_n^2, C = sum w ||u||^2;
 *   Dg[(s*N+t)*d+n] = A_n / (V_n + lambda) (0 where that denominator is 0),
 *   Ld[s*N+t] = max(0, C - 2 sum_n Dg_n A_n + sum_n Dg_n^2 V_n) / (C + 1e-12).
 *   Unobserved pairs: Dg = 0, Ld = 1e30.  Self pairs: Dg = 1, Ld = 0.  No clip.
 *   Outputs Dg [N, N, d] and Ld [N, N] float32 (rounded once).  lambda >= 0.
 *   ws: exfold_calibrate_workspace_size(layer, m, mode) bytes.
 */
exfold_status exfold_calibrate_diagonal(const exfold_layer *layer, const void *x_cal, int64_t m,
                                        double lambda, int32_t mode, float *Dg, float *Ld, void *ws,
                                        size_t ws_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* EXFOLD_H */
