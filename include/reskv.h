/*
 * reskv.h - C ABI of the ResKV hot path on AMD Instinct MI355X (gfx950).
 *
 * ResKV keeps, per (layer, KV head), a fixed budget of b = m + r cache slots:
 * m exact "main" tokens and r "residual" entries that summarise the evicted
 * tokens by a mean key, a mean value and a population count (Sec. 5.1-5.3 of
 * the paper). At decode, main tokens and residual entries share one softmax;
 * the residual logits carry log-count and a per-query dynamic gate (Sec. 5.4,
 * Sec. 5.5.2; App. D, Algorithm 2).
 *
 * One call handles one layer. All tensors are caller-owned device buffers
 * (row-major, innermost dimension last) unless a name ends in _host. The
 * library allocates nothing, keeps no pointer after a call returns, and
 * enqueues its kernels on the caller's HIP stream (passed as void*, i.e. a
 * hipStream_t; NULL is the null stream). Calls are asynchronous: argument
 * errors are reported by the return value before anything is launched;
 * faults inside a kernel surface at the caller's next synchronisation.
 * A call enqueues kernel launches only (no memset, copy, allocation or
 * synchronisation), and decode reads the cache lengths on the device, so
 * calls can be captured into a HIP graph and replayed; host arrays (_host)
 * are read when the call is made, i.e. at capture.
 *
 * Shapes: B = batch, Hq / Hkv = query / KV heads with Hq % Hkv == 0 and
 * G = Hq / Hkv <= 16 (grouped-query attention: query head h reads KV head
 * h / G, and the G heads of a group share its main indices and residual
 * entries, Sec. 6.1 and App. B), d = head_dim in {64, 128}, S = row stride
 * of the prefill K/V, C = slot capacity per (sequence, KV head), Rcap =
 * residual capacity.
 *
 * Cache layout per (b, kv head): slots [0, r) hold residual entries (mean
 * key / mean value, log-count in logc[0..r)); slots [r, r + main_len) hold
 * main tokens in ascending source position, followed by tokens appended
 * during decode. res_len[b*Hkv + h] = r, main_len[b*Hkv + h] = main slots.
 */
#ifndef RESKV_H
#define RESKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RESKV_OK = 0,
  RESKV_ERR_INVALID_ARG = 1,  /* shape, pointer or parameter out of range */
  RESKV_ERR_UNSUPPORTED = 2,  /* valid but not implemented (d, G, dtype) */
  RESKV_ERR_WORKSPACE = 3,    /* workspace missing or too small */
  RESKV_ERR_HIP = 4           /* a HIP runtime call failed at launch */
} reskv_status_t;

typedef enum { RESKV_F32 = 0, RESKV_BF16 = 1 } reskv_dtype_t;

typedef struct {
  int32_t batch;         /* B >= 1 */
  int32_t num_q_heads;   /* Hq, multiple of Hkv, Hq / Hkv <= 16 */
  int32_t num_kv_heads;  /* Hkv >= 1 */
  int32_t head_dim;      /* d: 64 or 128 */
  int32_t dtype;         /* reskv_dtype_t of every K/V/q tensor */
  int32_t slot_cap;      /* C: slots per (b, kv head) of kc, vc, main_idx */
  int32_t res_cap;       /* Rcap >= 1: entries per (b, kv head) of logc */
} reskv_shape_t;

typedef struct {
  int32_t max_seq_len;   /* S: row stride (in rows) of k and v */
  int32_t obs_window;    /* w: observation-window queries per q head, 1..S */
  int32_t recent_window; /* |P| before clamping to m: protected last tokens */
  int32_t lloyd_iters;   /* T >= 1: (assign, update) rounds, App. B.3 uses 4 */
  int32_t fit_rows;      /* leading window rows per q head that score, 1..w;
                            0 = all w. The validation proxy scores with the
                            fit part only (Sec. 5.5.1) */
  int32_t pool_kernel;   /* taps of the centred zero-padded score pooling,
                            odd, 1..31; 0 = 5. SnapKV (App. B.2.2) pools
                            with 5; H2O (w window queries, recent 64) and
                            TOVA (w = 1, recent 1) use 1 (App. B.2.2,
                            compared methods) */
} reskv_build_params_t;

typedef struct {
  const float* tau;      /* device [B*Hq] per-query threshold, or NULL */
  float tau_scalar;      /* threshold when tau == NULL (App. B.3: 0.25) */
  float alpha;           /* sigmoid slope 1/T_g (App. B.3: 12) */
  float g_min;           /* gate floor in [0, 1] (App. B.3: 0) */
  float beta;            /* log-count exponent (App. B.3: 1) */
} reskv_gate_t;

/*
 * reskv_build_cache - construct the main + residual cache of one layer from
 * its prefill K/V (App. D, Algorithm 1 with r given per (b, kv head)).
 *
 * Steps, per (b, kv head): observation-window scores (App. B.2.2: window
 * queries at positions s-w..s-1 attend causally, softmax per row, summed
 * over the G query heads, pool_kernel-tap (5 by default) zero-padded
 * pooling over the positions before the protected window; with fit_rows = f > 0 only the rows at
 * s-w..s-w+f-1 score, the fit part of Sec. 5.5.1); main selection
 * M = P u Top_{m-|P|}(scores) with ties to the lower position (Sec. 5.2,
 * main-selection equation);
 * Lloyd partition of the evicted set E = S \ M into r groups, seeded by the
 * evicted tokens ranked k_top..k_top+r-1 (Sec. 5.3, partition objective;
 * App. B.3); entries = (mean key, mean value, count) of the final groups
 * (Sec. 5.3, summary equation).
 *
 *   k, v            [B, Hkv, S, d]   prefill keys/values (rows >= s unused)
 *   seq_len_host    [B]              s per sequence, w <= s <= S
 *   q_obs           [B, Hq, w, d]    window queries (row i at position s-w+i)
 *   budget_host     [B]              b per KV head of sequence b, b <= C
 *   res_count_host  [B*Hkv]          r, 0 <= r < b, r <= Rcap
 *   kc, vc          [B, Hkv, C, d]   out: slots [0,r) residual, [r,r+m') main
 *   logc            [B, Hkv, Rcap]   out fp32: log c_j, -inf if group empty
 *   main_idx        [B, Hkv, C]      out int32: source positions of main
 *                                    slots, ascending; m' = min(m, s) valid
 *   res_len         [B*Hkv]          out int32: r
 *   main_len        [B*Hkv]          out int32: m' = min(b - r, s)
 *   dbg_scores      [B, Hkv, S]      optional (NULL): pooled scores, fp32
 *   dbg_assign      [T, B, Hkv, S]   optional (NULL): per Lloyd round, the
 *                                    group of each evicted position (-1 for
 *                                    main positions and rows >= s)
 *   dbg_centers     [T, B, Hkv, Rcap, d] optional (NULL), fp32: per Lloyd
 *                                    round, the centres that round assigns
 *                                    against (round 0: the seed keys; round
 *                                    t: the means of round t-1's groups, an
 *                                    empty group keeping its centre); rows
 *                                    j >= r' = min(r, |E|) are 0
 *   workspace       device scratch of reskv_build_workspace_size() bytes
 *
 * When s <= m every token is main and the r residual entries are empty.
 * Returns RESKV_OK or an error code before launching anything.
 */
reskv_status_t reskv_build_cache(const reskv_shape_t* shape,
                                 const reskv_build_params_t* params,
                                 const void* k, const void* v,
                                 const int32_t* seq_len_host,
                                 const void* q_obs,
                                 const int32_t* budget_host,
                                 const int32_t* res_count_host,
                                 void* kc, void* vc, float* logc,
                                 int32_t* main_idx,
                                 int32_t* res_len, int32_t* main_len,
                                 float* dbg_scores, int32_t* dbg_assign,
                                 float* dbg_centers,
                                 void* workspace, size_t workspace_bytes,
                                 void* stream);

/* Bytes of device workspace reskv_build_cache needs for these arguments
 * (0 if the arguments are invalid). The per-head sizes (s, b, r) fix the
 * grids and scratch of the construction, so the host arrays of the call
 * are arguments here too. */
size_t reskv_build_workspace_size(const reskv_shape_t* shape,
                                  const reskv_build_params_t* params,
                                  const int32_t* seq_len_host,
                                  const int32_t* budget_host,
                                  const int32_t* res_count_host);

/*
 * reskv_build_cache_adakv - construction with the top-k budget shared
 * across the KV heads of each sequence by AdaKV's cross-head allocation
 * (App. B.2.2, compared methods: AdaKV allocates the retained budget across
 * KV heads from the SnapKV scores, safeguard coefficient 0.2), followed by
 * the residual construction of reskv_build_cache.
 *
 * Per (b, kv head) the uniform split gives m = b - r, the protected window
 * |P| = min(recent_window, m, s) and the scored positions [0, s - |P|) with
 * k_top = m - |P|, exactly as reskv_build_cache. Heads with s <= m keep every
 * token and take no part. Among the others of sequence b:
 *   - head h keeps floor(safeguard * k_top_h) of its best-scored tokens
 *     (floor of the double product);
 *   - the remaining sum(k_top_h) - sum(floor) slots go down one ranking of
 *     every head's other scored tokens, by score descending, then KV head
 *     ascending, then position ascending; a head takes its next token only
 *     while it holds fewer than cap_h = min(s - |P|, C' - r_h - |P|) top-k
 *     tokens (a head can hold more than k_top_h, so slot_cap above the
 *     budget leaves room to grow), with C' = slot_cap - decode_reserve.
 * Head h then keeps its |P| recent tokens and its k'_h best-scored tokens
 * (ties to the lower position), and its r residual entries summarise the
 * rest as in reskv_build_cache (seeds: the evicted tokens of rank
 * k'_h .. k'_h + r - 1). safeguard = 1 gives the uniform split of
 * reskv_build_cache; safeguard = 0 is one top-k over all heads of a sequence.
 *
 *   safeguard       in [0, 1] (App. B.2.2: 0.2); Hkv <= 32
 *   decode_reserve  slots per (b, kv head) kept free for the tokens that
 *                   decode appends (Sec. 3.1): no head grows past
 *                   slot_cap - decode_reserve, so after construction every
 *                   head has room for decode_reserve appended tokens;
 *                   0 <= decode_reserve and budget[b] + decode_reserve <=
 *                   slot_cap
 *   other arguments as for reskv_build_cache, except:
 *   main_len        out int32 [B*Hkv]: |P| + k'_h (min(m, s) for heads with
 *                   s <= m); main_idx holds that many positions
 *   workspace       device scratch of reskv_build_adakv_workspace_size()
 *                   bytes (sized for the widest allocation of every head)
 * Returns RESKV_OK or an error code before launching anything.
 */
reskv_status_t reskv_build_cache_adakv(const reskv_shape_t* shape,
                                       const reskv_build_params_t* params,
                                       double safeguard,
                                       int32_t decode_reserve,
                                       const void* k, const void* v,
                                       const int32_t* seq_len_host,
                                       const void* q_obs,
                                       const int32_t* budget_host,
                                       const int32_t* res_count_host,
                                       void* kc, void* vc, float* logc,
                                       int32_t* main_idx,
                                       int32_t* res_len, int32_t* main_len,
                                       float* dbg_scores, int32_t* dbg_assign,
                                       float* dbg_centers,
                                       void* workspace, size_t workspace_bytes,
                                       void* stream);

/* Bytes of device workspace reskv_build_cache_adakv needs (0 if invalid). */
size_t reskv_build_adakv_workspace_size(const reskv_shape_t* shape,
                                        const reskv_build_params_t* params,
                                        double safeguard,
                                        int32_t decode_reserve,
                                        const int32_t* seq_len_host,
                                        const int32_t* budget_host,
                                        const int32_t* res_count_host);

typedef struct {
  const double* grid_host;  /* [n_grid] budget fractions f in [0, 1); at least
                               one is 0 (App. B.3: 0, .05, .10, .15, .20) */
  int32_t n_grid;           /* 1..8 */
  int32_t val_rows;         /* trailing window rows per q head held out for
                               validation, 1..w-1; the other w - val_rows
                               rows are the fit part (App. B.3: 8 of 32 at
                               G = 4, i.e. 96 fit and 32 validation queries) */
  float delta;              /* relative margin in [0, 1] (App. B.3: 0.01) */
} reskv_proxy_params_t;

/*
 * reskv_build_cache_proxy - construction with the residual count chosen per
 * (b, kv head) by the validation proxy (Sec. 5.5.1, validation-loss and
 * margin equations; App. D, Algorithm 1).
 *
 * The fit rows (the leading w - val_rows rows of every query head's
 * window) score the tokens once. For each grid fraction f the candidate
 * count is r_f = floor(f * b + 1/2) and the candidate cache is built as by
 * reskv_build_cache with res_count = r_f and fit_rows = w - val_rows. Every
 * validation query q (the trailing val_rows rows of the G heads of the
 * group, at their own window positions) is decoded against each candidate
 * with the decode rule of reskv_decode_attn (gate at gate->tau_scalar;
 * gate->tau is not read) and against the whole prefix [0, s) without
 * compression, o_S(q); the candidate's loss is the mean over the G *
 * val_rows queries of ||o_f(q) - o_S(q)||^2. With r* the count of least
 * loss among r_f > 0 (ties to the smaller count), r* is kept when
 * L(r*) < (1 - delta) * L(0), evaluated in fp32, else r = 0; the outputs
 * then hold that candidate's cache, exactly as reskv_build_cache writes it.
 *
 *   params          as for reskv_build_cache; fit_rows must be 0 or
 *                   w - val_rows
 *   k, v, seq_len_host, q_obs, budget_host   as for reskv_build_cache
 *   kc, vc, logc, main_idx, res_len, main_len  out, as for
 *                   reskv_build_cache with res_len = the chosen r
 *   val_loss        optional (NULL) out fp32 [B*Hkv, n_grid]: the loss of
 *                   every candidate, in grid order
 *   workspace       device scratch of reskv_build_proxy_workspace_size()
 *                   bytes; it holds every candidate cache
 *
 * Every candidate must satisfy r_f < b and r_f <= Rcap.
 * Returns RESKV_OK or an error code before launching anything.
 */
reskv_status_t reskv_build_cache_proxy(const reskv_shape_t* shape,
                                       const reskv_build_params_t* params,
                                       const reskv_proxy_params_t* proxy,
                                       const reskv_gate_t* gate,
                                       const void* k, const void* v,
                                       const int32_t* seq_len_host,
                                       const void* q_obs,
                                       const int32_t* budget_host,
                                       void* kc, void* vc, float* logc,
                                       int32_t* main_idx,
                                       int32_t* res_len, int32_t* main_len,
                                       float* val_loss,
                                       void* workspace, size_t workspace_bytes,
                                       void* stream);

/* Bytes of device workspace reskv_build_cache_proxy needs (0 if invalid). */
size_t reskv_build_proxy_workspace_size(const reskv_shape_t* shape,
                                        const reskv_build_params_t* params,
                                        const reskv_proxy_params_t* proxy,
                                        const int32_t* seq_len_host,
                                        const int32_t* budget_host);

/*
 * reskv_decode_attn - one decode step of shared-softmax attention for one
 * layer (Sec. 5.4: residual-logit, denominator, numerator and output
 * equations; Sec. 5.5.2: gate; App. D, Algorithm 2).
 *
 * For query head h of sequence b (KV head kv = h / G, r = res_len, n =
 * main_len):
 *   a_p   = <q, k_p> / sqrt(d)                           main slots
 *   p_max = max_p e^{a_p} / sum_p e^{a_p}
 *   g     = max(g_min, sigmoid((tau - p_max) * alpha))
 *   at_j  = <q, kbar_j> / sqrt(d) + beta * logc_j + log g  residual slots
 *   out   = (sum e^{a_p} v_p + sum e^{at_j} vbar_j) / (sum e^{a_p} + sum e^{at_j})
 * Entries with logc = -inf contribute nothing. main_len must be >= 1.
 *
 *   q               [B, Hq, d]       this step's queries
 *   kc, vc, logc    cache as written by reskv_build_cache / reskv_append_kv
 *   res_len, main_len  [B*Hkv] int32, read on the device
 *   k_new, v_new    [B, Hkv, d] optional (both or neither): this step's
 *                   token, appended as by reskv_append_kv before attending
 *                   (kc, vc and main_len are then written)
 *   out             [B, Hq, d] fp32
 *   dbg_lse_main    [B*Hq] optional: log sum_p e^{a_p}
 *   dbg_lse_res     [B*Hq] optional: log sum_j e^{<q,kbar_j>/sqrt(d) + beta logc_j}
 *   dbg_gate        [B*Hq] optional: g
 *   workspace       device scratch of reskv_decode_workspace_size() bytes
 *                   (split-K partials); calls sharing one must not overlap.
 *
 * Lengths read on the device are clamped to the capacities, so corrupt
 * lengths cannot make the kernels read outside the cache.
 *
 * Performance: the slot capacity C sets the head stride of kc and vc
 * (C * d * element bytes). With one block per (b, kv head) (from 256 pairs
 * on) every head is streamed at once, and a few strides put many heads on
 * the same HBM channels: at 256 heads of 2048 live slots, d = 128, bf16, a
 * call took 48-51 us at most capacities between 2056 and 2552 slots and up
 * to 57 us at the worst one measured (2064). The kernels accept any C; a
 * caller tuning for speed can time a few capacities at its own shape.
 */
reskv_status_t reskv_decode_attn(const reskv_shape_t* shape,
                                 const reskv_gate_t* gate,
                                 const void* q,
                                 void* kc, void* vc,
                                 const float* logc,
                                 const int32_t* res_len,
                                 int32_t* main_len,
                                 const void* k_new, const void* v_new,
                                 float* out,
                                 float* dbg_lse_main, float* dbg_lse_res,
                                 float* dbg_gate,
                                 void* workspace, size_t workspace_bytes,
                                 void* stream);

/* Bytes of device workspace reskv_decode_attn needs (0 if invalid or if
 * the capacities need more split-K partials than one block can merge). */
size_t reskv_decode_workspace_size(const reskv_shape_t* shape);

/*
 * reskv_decode_attn_ragged - reskv_decode_attn scheduled for batches whose
 * (b, kv head) caches differ widely in length (ragged contexts, budgets or
 * residual counts): the same computation (Sec. 5.4, Sec. 5.5.2, App. D,
 * Algorithm 2, with the optional fused append) and the same arguments, but
 * the work is split into 64-slot units over the whole batch (per head its
 * residual units, then its main units) and every block of the grid streams
 * an equal range of that list, so no compute unit waits on the longest
 * head. Heads that span several blocks are merged by a second kernel, which
 * also advances main_len. Outputs equal reskv_decode_attn's within rounding
 * (a different order of the same fp32 sums).
 *
 *   workspace       device scratch of reskv_decode_ragged_workspace_size()
 *                   bytes (the per-call plan and the partial records of
 *                   shared heads); calls sharing one must not overlap.
 * Supported: G <= 8, B*Hkv <= 2048, C <= 64960 slots, bf16 rows (fp32
 * rows of d = 64); otherwise RESKV_ERR_UNSUPPORTED. Errors as for
 * reskv_decode_attn.
 */
reskv_status_t reskv_decode_attn_ragged(const reskv_shape_t* shape,
                                        const reskv_gate_t* gate,
                                        const void* q,
                                        void* kc, void* vc,
                                        const float* logc,
                                        const int32_t* res_len,
                                        int32_t* main_len,
                                        const void* k_new, const void* v_new,
                                        float* out,
                                        float* dbg_lse_main, float* dbg_lse_res,
                                        float* dbg_gate,
                                        void* workspace, size_t workspace_bytes,
                                        void* stream);

/* Bytes of device workspace reskv_decode_attn_ragged needs (0 if invalid or
 * unsupported). */
size_t reskv_decode_ragged_workspace_size(const reskv_shape_t* shape);

/*
 * reskv_decode_attn_static - reskv_decode_attn without a workspace, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation). Same arguments,
 * results and kernels as reskv_decode_attn; the split-K records live in a
 * scratch array of 16 MiB that the library holds in device memory on every
 * GPU it runs on until the process ends. The call allocates nothing.
 *
 *   stream          must belong to the calling thread's current device (the
 *                   scratch of that device is used)
 * Errors: RESKV_ERR_WORKSPACE when the shape takes the split-K path (fewer
 * than 256 (sequence, KV head) pairs, or fp32 rows of 128) and its records
 * need more than 16 MiB (reskv_decode_workspace_size(shape) > 16 MiB);
 * otherwise as for reskv_decode_attn. All calls on one GPU share its scratch: calls that
 * overlap in time on one GPU (on different streams) race and must not be
 * issued; calls ordered on one stream are safe.
 */
reskv_status_t reskv_decode_attn_static(const reskv_shape_t* shape,
                                        const reskv_gate_t* gate,
                                        const void* q,
                                        void* kc, void* vc,
                                        const float* logc,
                                        const int32_t* res_len,
                                        int32_t* main_len,
                                        const void* k_new, const void* v_new,
                                        float* out,
                                        float* dbg_lse_main, float* dbg_lse_res,
                                        float* dbg_gate,
                                        void* stream);

/*
 * reskv_decode_branches - the two branches of one decode step, each under
 * its own softmax: the form in which a fused main-branch attention kernel
 * and a separately evaluated residual branch are combined through
 * log-sum-exp statistics (Sec. 6.1 implementation notes). With a_p and the
 * gate g as for reskv_decode_attn and at_j = <q, kbar_j>/sqrt(d) +
 * beta * logc_j (no gate):
 *   out_main = sum_p e^{a_p} v_p / sum_p e^{a_p},   lse_main = log sum_p e^{a_p}
 *   out_res  = sum_j e^{at_j} vbar_j / sum_j e^{at_j}, lse_res = log sum_j e^{at_j}
 * (out_res = 0 and lse_res = -inf when no entry is populated).
 *
 *   q, kc, vc, logc, res_len, main_len  as for reskv_decode_attn (no append)
 *   out_main, out_res   [B, Hq, d] fp32
 *   lse_main, lse_res, gate_out  [B*Hq] fp32
 *   workspace           reskv_decode_workspace_size() bytes
 * Returns RESKV_OK or an error code before launching anything.
 */
reskv_status_t reskv_decode_branches(const reskv_shape_t* shape,
                                     const reskv_gate_t* gate,
                                     const void* q,
                                     const void* kc, const void* vc,
                                     const float* logc,
                                     const int32_t* res_len,
                                     const int32_t* main_len,
                                     float* out_main, float* lse_main,
                                     float* out_res, float* lse_res,
                                     float* gate_out,
                                     void* workspace, size_t workspace_bytes,
                                     void* stream);

typedef enum {
  RESKV_MERGE_SHARED = 0,   /* log-sum-exp merge: the shared softmax */
  RESKV_MERGE_SEPARATE = 1  /* separate normalisations mixed by the gate */
} reskv_merge_mode_t;

/*
 * reskv_merge_branches - combine the outputs of reskv_decode_branches.
 *   RESKV_MERGE_SHARED: out = (e^{lse_main} out_main + g e^{lse_res} out_res)
 *     / (e^{lse_main} + g e^{lse_res}), which is reskv_decode_attn's output
 *     (Sec. 5.4 output equation over branch statistics, Sec. 6.1).
 *   RESKV_MERGE_SEPARATE: out = (1 - g) out_main + g out_res, g taken as 0
 *     where lse_res = -inf: the ablation without the shared softmax
 *     (Sec. 6.6 ablation table; the paper gives no formula, this mixture is
 *     this library's reading of it).
 * All arrays fp32 on the device, shapes as for reskv_decode_branches; out
 * [B, Hq, d] may alias neither input.
 */
reskv_status_t reskv_merge_branches(const reskv_shape_t* shape, int32_t mode,
                                    const float* out_main, const float* lse_main,
                                    const float* out_res, const float* lse_res,
                                    const float* gate, float* out,
                                    void* stream);

/*
 * reskv_append_kv - append one decode token per (b, kv head) as a main slot
 * (Sec. 3.1: each decode step appends the new token's key and value).
 * Writes k_new/v_new [B, Hkv, d] into slot res_len + main_len and increments
 * main_len, on the device. A (b, kv head) whose cache is full (res_len +
 * main_len == C) is left unchanged.
 */
reskv_status_t reskv_append_kv(const reskv_shape_t* shape,
                               const void* k_new, const void* v_new,
                               void* kc, void* vc,
                               const int32_t* res_len, int32_t* main_len,
                               void* stream);

/* Static description of a status code. */
const char* reskv_status_string(reskv_status_t status);

/* Detail of the last error returned on the calling thread ("" if none). */
const char* reskv_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* RESKV_H */
