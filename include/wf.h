/*
 * wf.h -- C-ABI of libwf: wavefront decoding and encoding of a spatial
 * autoregressive context model on one MI355X (gfx950) GPU.
 *
 * The method (Murai et al., "Wavefront Parallelization for Efficient Learned
 * Image Compression"): the latents of an H x W grid form a DAG whose edges are
 * the causal taps of a 5x5 masked convolution (Sec. III-A, Eq. 3; Appendix A,
 * Def. 1).  The linear rank t(i,j) = lambda*i + j with the smallest shear
 * lambda that satisfies the hyperplane condition (Sec. III-B, Eq. 5-7) is a
 * valid schedule with W + lambda*(H-1) steps, optimal when W >= lambda
 * (Appendix A, Thm. 1).  On a narrower grid (W < lambda) every latent
 * depends on its raster predecessor, so the earliest-possible schedule is the
 * raster order itself: the shear W, H*W steps.  All latents of one step (a wavefront) are decoded
 * together: their causal taps are gathered from the reconstruction
 * (Sec. III-C, selective im2col), the masked-conv context and the 1x1
 * entropy-parameter network are evaluated as batched products, and the
 * reconstruction y_hat is written before the next step starts.
 *
 * Conventions for every entry point:
 *  - Return value: WF_OK (0) or a negative wf_status; wf_last_error() then
 *    holds a message for the calling thread.  No exception crosses the ABI.
 *  - Arguments are validated before any work is enqueued; a rejected call
 *    changes nothing.
 *  - "host" pointers are read during the call only; "device" pointers must
 *    stay valid until the enqueued work on the given stream has finished.
 *  - All arrays are dense, row-major, NHWC (channel innermost).
 */
#ifndef WF_H
#define WF_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    WF_OK = 0,
    WF_E_INVALID = -1,      /* bad argument (NULL, non-positive size, ...)     */
    WF_E_UNSUPPORTED = -2,  /* valid but not supported by this library         */
    WF_E_HIP = -3,          /* a HIP runtime call failed                       */
    WF_E_NOMEM = -4,        /* device or host allocation failed                */
    WF_E_TIMEOUT = -5,      /* a device-side wait exceeded its spin budget     */
    WF_E_STREAM = -6,       /* a malformed rANS stream (decode from streams)   */
    WF_E_CAPACITY = -7      /* encoded streams larger than the caller's buffer */
} wf_status;

/* Entropy coder of the symbols (wf_desc.entropy_coder). */
typedef enum {
    WF_EC_NONE = 0,         /* symbols are passed as int32 arrays                      */
    WF_EC_RANS = 1          /* also wf_encode_bits / wf_decode_bits: rANS streams (K = 1:
                               the Gaussian coder, K = 3: the mixture coder), stream or
                               graph driver, exact decode (group <= 1)                   */
} wf_entropy_coder;

/* Causal masks (Def. 1: a (2R+1)x(2R+1) kernel keeps the R rows above within
 * horizontal offset R, and the R latents to the left; least shear R + 1). */
typedef enum {
    WF_MASK_FULL = 0,       /* 5x5, 12 taps: rows -2,-1 with dx in [-2,2]; (0,-2), (0,-1); lambda = 3 */
    WF_MASK_RELAXED = 1,    /* 5x5, 10 taps: the full mask without (-1,+2) and (-2,+2); lambda = 2   */
    WF_MASK_3X3 = 2,        /* 3x3, 4 taps: row -1 with dx in [-1,1]; (0,-1); lambda = 2            */
    WF_MASK_7X7 = 3         /* 7x7, 24 taps: rows -3..-1 with dx in [-3,3]; (0,-3..-1); lambda = 4  */
} wf_mask;

/* Operand precision of every product (the paper fixes none; fp32 is the
 * reference).  WF_BF16 runs every product on bf16 MFMA with fp32 accumulation:
 * weights are rounded to bf16 (round to nearest even); each activation (taps,
 * hyperprior params, context, hidden vectors) is carried as the pair
 * hi = bf16(x), lo = bf16(x - hi), about 2^-17 relative, so the weights are
 * the only coarse rounding.  Needs M a multiple of 32. */
typedef enum {
    WF_FP32 = 0,            /* fp32 operands, fp32 accumulate                           */
    WF_BF16 = 1             /* bf16 weights, bf16-pair activations, fp32 accumulate     */
} wf_precision;

typedef enum {
    WF_DRIVER_STREAM = 0,   /* per-step kernel launches, enqueued one by one on the stream */
    WF_DRIVER_GRAPH = 1,    /* the same per-step kernels, replayed from one HIP graph      */
    WF_DRIVER_PERSISTENT = 2,/* one cooperative kernel, device-wide barrier per phase      */
    WF_DRIVER_DATAFLOW = 3, /* one cooperative kernel; every job waits only for the jobs it
                               depends on (per-step, per-row-tile completion counters)     */
    WF_DRIVER_RESIDENT = 4  /* one cooperative kernel, two workgroups per compute unit, each
                               holding one slice of the weights in registers for the whole
                               decode (an old-tap context k-part, a layer-1/-2 column tile
                               or a layer-3 channel tile) and running that slice's product
                               for every 16-row band of every step, as soon as the bands it
                               reads are complete (per-task completion counters).
                               WF_E_UNSUPPORTED when the slices do not fit the registers
                               or the compute units, M is not a multiple of 32 or the
                               schedule has more than 4095 steps; calls need y_hat
                               aligned to 128 bytes (WF_E_INVALID otherwise).  fp32:
                               layer-1 and -2 outputs are read until no value holds an
                               all-ones fill word, a NaN that finite inputs never yield;
                               inputs holding NaNs with that exact bit pattern can make
                               a call end in WF_E_TIMEOUT (after the wait budget of
                               wf_plan_set_waits) instead of returning NaNs               */
} wf_driver;

/* Block order of the last layer's output rows (w3, b3).  The kernels use the
 * native order; a checkpoint whose entropy-parameter head emits the scales
 * first is imported by naming its order here (the plan permutes the rows). */
typedef enum {
    WF_ORDER_NATIVE = 0,       /* K = 1: mean | scale;  K = 3: weight | mean | scale */
    WF_ORDER_SCALES_FIRST = 1  /* K = 1: scale | mean;  K = 3: scale | mean | weight */
} wf_param_order;

/*
 * Model and problem description.  All weight arrays are HOST memory in
 * PyTorch layouts and are copied (and repacked) by wf_plan.
 *   ctx_w [2M][M][k][k]  masked conv weight, k = 5 (3, 7 for WF_MASK_3X3 / _7X7);
 *                        masked positions are ignored
 *   ctx_b [2M]
 *   w1 [d1][4M], b1 [d1]   layer 1 input is [psi (2M) ; ctx (2M)]
 *   w2 [d2][d1], b2 [d2]
 *   w3 [n3][d2], b3 [n3]   n3 = 2M for K = 1 (rows: mean | scale),
 *                          n3 = 9M for K = 3 (rows: weight | mean | scale,
 *                          each block component-major: block*3M + k*M + c);
 *                          with param_order = WF_ORDER_SCALES_FIRST the blocks
 *                          come in the order scale | mean (| weight)
 *   scale_table [L]        strictly increasing, positive
 * Hidden layers use LeakyReLU with slope lrelu_slope; the last layer is linear.
 */
typedef struct {
    int32_t H, W;           /* latent rows and columns                              */
    int32_t M;              /* latent channels; multiple of 16                       */
    int32_t B;              /* images decoded together on one wavefront sweep        */
    int32_t K;              /* 1: mean-scale Gaussian; 3: 3-component mixture        */
    int32_t d1, d2;         /* hidden widths of the entropy-parameter network        */
    int32_t mask;           /* wf_mask                                               */
    int32_t precision;      /* wf_precision                                          */
    int32_t driver;         /* wf_driver                                             */
    float lrelu_slope;
    const float *ctx_w, *ctx_b;
    const float *w1, *b1, *w2, *b2, *w3, *b3;
    const float *scale_table;
    int32_t L;              /* table length, 2 <= L <= 256                            */
    int32_t group;          /* context approximation (Sec. III-D, Fig. 3): 0 or 1 decodes
                               exactly; N > 1 decodes N consecutive wavefronts as one
                               step, each tap in the latent's own group replaced, channel
                               by channel, by the mean of its decoded in-image taps (zero
                               when none is decoded).  N > 1 needs the stream or graph
                               driver (WF_E_UNSUPPORTED otherwise).                      */
    int32_t param_order;    /* wf_param_order: block order of the rows of w3 and b3        */
    int32_t entropy_coder;  /* wf_entropy_coder                                             */
    int32_t cu_limit;       /* 0: plan the in-launch drivers (persistent, dataflow,
                               resident) for every compute unit; N > 0: for at most N
                               (a plan that then cannot be resident is refused with
                               WF_E_UNSUPPORTED)                                        */
} wf_desc;

/*
 * Per-call outputs, all DEVICE memory owned by the caller.
 *   y_hat     [B][H][W][M]     reconstruction (s + mean); also the AR state
 *   mean      [B][H][W][M]     dequantisation offset (mixture mean for K = 3)
 *   scale     [B][H][W][K][M]  max(raw scale, scale_table[0])
 *   idx       [B][H][W][K][M]  #{l in [0, L-2] : scale_table[l] < scale}
 *   weight    [B][H][W][K][M]  mixture weights (K = 3 only; NULL for K = 1)
 *   comp_mean [B][H][W][K][M]  component means (K = 3 only; NULL for K = 1)
 */
typedef struct {
    float *y_hat, *mean, *scale;
    int32_t *idx;
    float *weight, *comp_mean;
} wf_out;

typedef struct wf_plan_s *wf_plan_t;

/*
 * Schedule of an H x W grid under a mask (host only; no GPU needed).  This is
 * the exact schedule; wf_plan_schedule gives a plan's decoding steps, which
 * are groups floor(t / N) under context approximation.
 * Writes step_of[i*W + j] = lambda*i + j (HOST array of H*W int32, may be
 * NULL) and *n_steps = W + lambda*(H-1), where lambda is the least integer
 * shear with lambda*di + dj > 0 for every dependence vector of the mask
 * (Sec. III-B, Eq. 6-7), or W when W is smaller (the raster order, which is
 * then the earliest-possible schedule).  Also writes *lambda_out when
 * non-NULL.
 * Errors: WF_E_INVALID for H < 1, W < 1, an unknown mask or a NULL n_steps.
 */
int wf_schedule(int32_t H, int32_t W, int32_t mask, int32_t *step_of,
                int32_t *n_steps, int32_t *lambda_out);

/*
 * Validate a description without touching the GPU.  Returns WF_OK or the
 * error wf_plan would return for it before allocating anything.
 */
int wf_validate(const wf_desc *desc);

/*
 * Build a plan: schedule and step lists, weights repacked into the kernels'
 * tile layouts on the device, the scale table, the workspace, and (for the
 * graph driver) the instantiated graph.  Synchronous; uses the current HIP
 * device.  On success *out owns all of it until wf_plan_destroy.
 * The schedule is the linear rank of Sec. III-B (Eq. 5-7) with its step
 * lists (the wavefronts of Sec. III-A, Eq. 4; Appendix A, Thm. 1); the
 * weights are those of the masked-conv context model and the entropy-
 * parameter network of Sec. II-B (Eq. 1).
 * Errors: those of wf_validate; WF_E_NOMEM / WF_E_HIP when a device
 * allocation or copy fails (nothing is left allocated).
 */
int wf_plan(const wf_desc *desc, wf_plan_t *out);

/* Copy the plan's schedule out (HOST array of H*W int32): the decoding step
 * of every latent (its wavefront t, or its group floor(t / N) under context
 * approximation) and the number of steps. */
int wf_plan_schedule(wf_plan_t plan, int32_t *step_of, int32_t *n_steps);

/*
 * Race checking (host only; no device is touched): the dependency structure
 * that the in-launch drivers' kernels follow for the plan `desc` describes,
 * computed by the same functions the kernels call.  The causality of the
 * wavefront decode (Sec. III-A, Eq. 3-4: a latent is decoded after every
 * latent of its mask) then rests on these waits, which the test suite checks
 * by simulation.  desc->driver selects the layout of `out` (int32):
 *   WF_DRIVER_DATAFLOW: per job of the plan's job lists, in list order,
 *     {t, kind (0 CTX, 1 CTXL, 2 A, 3 B, 4 C0, 5 C1), part, row tile,
 *     column tile, list (0-7 critical, 8-15 context, by column tile mod 8),
 *     position in the global order, number of waits, then three waits
 *     (counter group, column tiles lo, hi, multiplicity)}: a wait holds
 *     until, for every class x, the group's counter of class x reaches the
 *     multiplicity times the number of column tiles in [lo, hi) of class x.
 *     A finished job bumps the counter of its class (column tile mod 8) in
 *     group (t*6 + kind)*(nrt_max + 1) + row tile and, for C0 and C1, in
 *     group (t*6 + kind)*(nrt_max + 1) + nrt_max.  The last entry is nrt_max.
 *   WF_DRIVER_RESIDENT: per task (step t, image b, 16-row band beta) in the
 *     global order, {t, b, beta, then for each role (0 CTX, 1 CTXL, 2 A, 3 B,
 *     4 C0, 5 C1, 6 H: the in-launch hoist of bf16 plans) three waits
 *     (role, task), role -1 for none}, as planned with the context parts
 *     before the last taking the taps older than two steps.
 * *needed receives the number of entries; out (HOST, capacity entries) may
 * be NULL.  Errors: WF_E_INVALID (desc, needed, capacity),
 * WF_E_UNSUPPORTED (another driver; any plan the driver refuses).
 */
int wf_plan_deps(const wf_desc *desc, int32_t *out, int64_t capacity, int64_t *needed);

/*
 * The bounded waits of the in-launch drivers (persistent, dataflow,
 * resident), for the calls after this one: spin_budget_ticks is the longest
 * one wait may spin, in ticks of the 100 MHz wall clock (<= 0: the default,
 * 1 s).  A wait past its budget, or one that sees an error recorded by
 * another workgroup, leaves the kernel, so the grid always drains and the
 * next wf_plan_sync returns WF_E_TIMEOUT; the next call starts afresh.
 * stall = 1 (for tests of that path) makes every counter and barrier wait
 * unreachable, so the calls time out by construction; stall = 0 restores
 * them.  The stream and graph drivers do not wait and ignore both.
 * Errors: WF_E_INVALID (NULL plan, stall not 0 or 1).
 */
int wf_plan_set_waits(wf_plan_t plan, int64_t spin_budget_ticks, int32_t stall);

/*
 * Coherence litmus test of the exchange inside one launch that the
 * persistent, dataflow and resident drivers rely on (the causality of
 * Sec. III-A, Eq. 4 across workgroups): `pairs` producer workgroups each
 * store `rounds` blocks of 1024 words with agent-coherent stores, wait for
 * them to land and bump a per-block counter (relaxed, agent scope); as many
 * consumer workgroups, each reading the blocks of a producer dealt to
 * another XCD, poll the counter (bounded, 1 s) and check every word.
 * mode 0: agent-coherent loads (buffers reused within a launch); mode 1:
 * ordinary cached loads of addresses written once per launch; mode 2: the
 * producer bumps the counter once its stores are issued (no wait for them
 * to land), the blocks start filled with an all-ones word, and the consumer
 * reads agent-coherent, reading again each word that still holds the fill
 * (bounded, 1 s) -- the resident driver's fp32 layer-1 and -2 outputs.
 * *mismatches receives the number of words read wrong (0 when the exchange
 * is coherent).  Synchronous (returns after the kernel finished on
 * `stream`).  Errors: WF_E_INVALID, WF_E_UNSUPPORTED (more workgroups than
 * can be resident), WF_E_NOMEM, WF_E_TIMEOUT (a consumer waited too long).
 */
int wf_litmus(int32_t mode, int32_t pairs, int32_t rounds, uint64_t *mismatches, hipStream_t stream);

/*
 * Decode (Sec. III-A, Eq. 2 evaluated in the wavefront order of Eq. 4; the
 * per-step batched gather and products of Sec. III-C): for every step
 * t = 0..T-1 and every latent on wavefront t, compute the parameters from the
 * already written y_hat and write y_hat = (float)sym + mean (Sec. II-A).
 *   psi [B][H][W][2M] DEVICE fp32 hyperprior parameters
 *   sym [B][H][W][M]  DEVICE int32 symbols
 * Asynchronous on `stream`; one call in flight per plan (the plan's
 * workspace is shared by its calls).
 */
int wf_decode(wf_plan_t plan, const float *psi, const int32_t *sym,
              const wf_out *out, hipStream_t stream);

/*
 * Encode (the quantiser of Sec. II-A run in the same wavefront order, so the
 * encoder sees exactly the context the decoder will): as decode, but the
 * symbol is sym_out = rint(y - mean) (fp32 subtract, round half to even) and
 * y_hat = (float)sym_out + mean.
 *   y       [B][H][W][M] DEVICE fp32 latents
 *   sym_out [B][H][W][M] DEVICE int32
 */
int wf_encode(wf_plan_t plan, const float *psi, const float *y, int32_t *sym_out,
              const wf_out *out, hipStream_t stream);

/*
 * Entropy coding with rANS (plans built with entropy_coder = WF_EC_RANS).
 * The entropy model is the discretised Gaussian of the symbol's scale level
 * (Sec. II-A; the paper pairs the wavefront decode with rANS, Sec. III-C).
 * Per level l, with T_l the level's table value: support n_l =
 * max(1, ceil(6 T_l)), symbols -n_l..n_l and an escape for |s| > n_l whose
 * excess follows in 15-bit chunks; frequencies in units of 2^-16,
 * f = 1 + floor(p (2^16 - 2 n_l - 2)) for the Gaussian mass p of
 * [s - 1/2, s + 1/2], the remainder added to s = 0.  Coder: 64-bit state in
 * [2^31, 2^63), 32-bit words.
 * K = 3 (the 3-component mixture): a symbol is coded with the mixture of its
 * channel's three Gaussians around the mixture mean, with frequencies built
 * in integer arithmetic from quantised parameters: weights
 * v_k = 1 + floor(4093 w_k) (the rest of 4096 to the largest), offsets
 * q_k = rint(16 (mu_k - mu)) in sixteenths of a symbol (within +-2^14), and
 * per level an integer CDF on sixteenths, G_l(x) = floor(2^20 Phi(x / (16 T_l))
 * + 1/2) for |x| < X_l = 16 (n_l + 1) (0 and 2^20 beyond).  With
 * F(s) = sum_k v_k G_{l_k}(16 s + 8 - q_k), symbols s_lo..s_hi that cover
 * every component's table and S of them, cum(s) = (s - s_lo) +
 * floor(F(s - 1) (2^16 - S - 1) / 2^32); the last slot (frequency 1) is the
 * escape, whose excess follows in 15-bit chunks.
 * Streams: one per (image b, grid row i, channel c), index k = (b*H + i)*M + c,
 * holding the row's symbols in column order (one per wavefront step); stream
 * k occupies words [offsets[k], offsets[k+1]) of `bits`: the final state
 * (high, low word) and then the renormalisation words in decoding order.
 *
 * wf_ec_tables (host only): the frequency tables of a scale table:
 * n[L], base[L+1] (first cumulative entry of each level), and, when cum is
 * non-NULL, the cumulative frequencies (base[L] entries, 2 n_l + 3 per level,
 * from 0 to 2^16).  Errors: WF_E_INVALID (NULL table, L outside [2, 256],
 * cum_cap < base[L]); WF_E_UNSUPPORTED when a level needs n_l > 16383.
 */
int wf_ec_tables(const float *scale_table, int32_t L, int32_t *n, int64_t *base,
                 uint32_t *cum, int64_t cum_cap);

/*
 * wf_mix_tables (host only): the mixture coder's level tables of a scale
 * table (K = 3; the CDFs G_l above): X[L], base[L+1] (first entry of each
 * level) and, when G is non-NULL, G_l(x) for x = -X_l..X_l at
 * base[l] + x + X_l (base[L] entries).  Errors as for wf_ec_tables.
 */
int wf_mix_tables(const float *scale_table, int32_t L, int32_t *X, int64_t *base,
                  uint32_t *G, int64_t G_cap);

/*
 * Encode (as wf_encode) and code the symbols into rANS streams.
 *   bits     DEVICE uint32, bits_capacity words
 *   offsets  DEVICE uint32 [B*H*M + 1]; offsets[B*H*M] = total words
 * The total is always written; when it exceeds bits_capacity nothing is
 * written to bits and the next wf_plan_sync returns WF_E_CAPACITY.
 * Asynchronous on `stream`.
 */
int wf_encode_bits(wf_plan_t plan, const float *psi, const float *y, int32_t *sym_out,
                   const wf_out *out, uint32_t *bits, int64_t bits_capacity,
                   uint32_t *offsets, hipStream_t stream);

/*
 * Decode with every symbol read from its rANS stream inside the step loop:
 * at the step of latent (b,i,j) the symbol of each channel c is decoded from
 * stream (b*H + i)*M + c at the latent's scale level (K = 3: under the
 * mixture of its three components), then y_hat = symbol + mean.  sym_out [B][H][W][M] (DEVICE int32) receives the
 * decoded symbols.  `bits` (DEVICE, n_words words) and `offsets` (DEVICE
 * [B*H*M + 1]) are as written by wf_encode_bits.  Reads never go past a
 * stream's end or n_words; a malformed stream makes the next wf_plan_sync
 * return WF_E_STREAM (the outputs are then unspecified).  Asynchronous.
 */
int wf_decode_bits(wf_plan_t plan, const float *psi, const uint32_t *bits, int64_t n_words,
                   const uint32_t *offsets, int32_t *sym_out, const wf_out *out,
                   hipStream_t stream);

/*
 * wf_decode for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same decode and outputs, but the call's working memory -- the hoisted
 * hyperprior half of layer 1 for every latent, the per-step activations, the
 * old-tap context parts, the bf16 pair copy of y_hat and the call's pointer
 * block -- lives in a static device array of the library (32 MiB, held by
 * every device the library runs on until the process ends) instead of the
 * plan's workspace.  It runs the stream driver's per-step kernels on `stream`
 * whatever the plan's driver, and calls no allocating routine.
 * Errors: as wf_decode; WF_E_UNSUPPORTED (with the bytes needed) when the
 * working memory exceeds 32 MiB (e.g. the 1920x1080 GMM workload needs about
 * 22 MB; the 3840x2160 M = 320 one does not fit).
 * All calls on one device share the array: calls that overlap on a device
 * (concurrent streams or threads) race and must be serialised by the caller.
 * No part of the array needs clearing: every element a call reads was
 * written earlier in the same call.
 */
int wf_decode_noalloc(wf_plan_t plan, const float *psi, const int32_t *sym, const wf_out *out,
                      hipStream_t stream);

/*
 * Measurement hook of the persistent, dataflow and resident drivers
 * (WF_E_UNSUPPORTED for the others).  With `stamps` non-NULL (DEVICE int64 array of `capacity`
 * entries) every later call records the device wall clock (100 MHz ticks):
 *  - persistent: at each device-wide barrier k = 0, 1, ...: entry k*(G+1) + g
 *    is the time workgroup g arrived at barrier k, entry k*(G+1) + G the time
 *    workgroup 0 left it.  A call has 2 + 3*T barriers (two before the first
 *    step, then one after each of a step's three phases), with either
 *    precision.
 *  - dataflow: three entries per job, 3*j + {0, 1, 2} = the time the job's
 *    workgroup started waiting for its inputs, the time they were complete,
 *    and the time its results had landed; j is the job's position in the
 *    plan's job lists (XCD classes 0..7 in turn, each in its topological order).
 *  - resident: three entries per task k (global order) and workgroup g,
 *    3*(k*G + g) + {0, 1, 2}: the times g started waiting for the task's
 *    inputs, found them complete and had its results published (0 where g's
 *    role and replica do not run task k); workgroups are in role order (the
 *    context parts, the last part, layers 1, 2, 3 mean and scale columns, the
 *    in-launch hoist).
 * G is the grid size written to *grid; *needed receives the entries a call
 * takes (either output may be NULL).  Entries past `capacity` are not
 * written.  stamps == NULL turns recording off.  The array stays owned by
 * the caller and must outlive the calls that record into it.
 */
int wf_plan_trace(wf_plan_t plan, int64_t *stamps, int64_t capacity, int64_t *needed,
                  int32_t *grid);

/*
 * Latency floor of one dependent step hop on the current device, measured
 * synchronously on a private stream: *node_us is the per-node time of a chain
 * of 512 empty kernels replayed from a HIP graph, *barrier_us the time of one
 * empty round of the persistent driver's device-wide barrier over its grid
 * (-1 when that grid cannot be resident).  Measurement support for the
 * latency-aware roofline; it touches no plan state except the device error
 * word (a barrier timeout is recorded there as for a call).
 */
int wf_measure_floor(wf_plan_t plan, float *node_us, float *barrier_us);

/*
 * Wait for `stream` and report a device-side error recorded by the plan's
 * kernels (WF_E_TIMEOUT when a bounded device-wide wait gave up, WF_E_STREAM
 * for a malformed rANS stream, WF_E_CAPACITY when encoded streams did not
 * fit).  Clears the recorded error.
 */
int wf_plan_sync(wf_plan_t plan, hipStream_t stream);

/*
 * The transforms around the autoregressive decode, for an end-to-end decode
 * timing (the latent pipeline of Sec. II-A; random weights, as no trained
 * ones are used): the hyper-decoder h_s (z_hat -> psi, the hyperprior half
 * of the entropy parameters) and the synthesis transform g_s (y_hat ->
 * image).  Layers (the mean-scale hyperprior model family the workloads are
 * named after; PyTorch weight layouts, HOST arrays copied by the plan):
 *   h_s: hs_w[0] [N][M][5][5]      transposed conv 5x5 s2 (padding 2, output
 *                                  padding 1), + hs_b[0] [M], ReLU
 *        hs_w[1] [M][3M/2][5][5]   the same, + hs_b[1], ReLU
 *        hs_w[2] [2M][3M/2][3][3]  conv 3x3 s1 (padding 1), + hs_b[2] [2M]
 *   g_s: gs_w[k] [Cin][Cout][5][5] transposed conv 5x5 s2 + gs_b[k], for
 *        (Cin, Cout) = (M, N), (N, N), (N, N), (N, 3); after each of the first
 *        three: inverse GDN, out_c = x_c sqrt(gdn_beta[k][c] +
 *        sum_j gdn_gamma[k][c][j] x_j^2)
 * z_hat has ceil(H/4) x ceil(W/4) pixels; psi is the top-left H x W of h_s's
 * output.  N, M and 3M/2 must be multiples of 16 (fp32) or 32 (bf16).
 */
typedef struct {
    int32_t N, M;           /* channels of z_hat and of y_hat                       */
    int32_t B, H, W;        /* images and the latent grid of y_hat                  */
    int32_t precision;      /* wf_precision (bf16: bf16 weights, activations as pairs) */
    const float *hs_w[3], *hs_b[3];
    const float *gs_w[4], *gs_b[4];
    const float *gdn_beta[3], *gdn_gamma[3];
} wf_xform_desc;

typedef struct wf_xform_s *wf_xform_t;

/* Build the transform plan (packed weights and workspace, ~2 x B*64*H*W*N
 * floats).  Synchronous; errors as wf_plan (WF_E_UNSUPPORTED for channel
 * counts off the k-block or activations beyond the 2 GiB buffer window). */
int wf_xform_plan(const wf_xform_desc *desc, wf_xform_t *out);

/* psi [B][H][W][2M] = h_s(z_hat [B][ceil(H/4)][ceil(W/4)][N]); DEVICE fp32,
 * asynchronous on `stream`, one call in flight per plan. */
int wf_hyper_synthesis(wf_xform_t plan, const float *z_hat, float *psi, hipStream_t stream);

/* image [B][16H][16W][3] = g_s(y_hat [B][H][W][M]); DEVICE fp32, asynchronous. */
int wf_synthesis(wf_xform_t plan, const float *y_hat, float *image, hipStream_t stream);

/* Release a transform plan.  NULL is ignored. */
void wf_xform_destroy(wf_xform_t plan);

/* Release everything the plan owns.  NULL is ignored. */
void wf_plan_destroy(wf_plan_t plan);

/* Message of the last failed call on this thread ("" if none). */
const char *wf_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* WF_H */
