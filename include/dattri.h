/*
 * dattri.h -- C ABI of the MI355X (gfx950) projected-gradient attribution
 * library (libdattri.so).
 *
 * The library computes, for a batch of examples and a set of linear layers,
 * each example's projected weight gradient per layer, concatenates the layer
 * blocks into one feature vector phi per example, and scores query features
 * against training features.  Definitions (paper sections):
 *
 *   - Sec. 3.2, Eq. (1): for one example with T token positions, the weight
 *     gradient of a linear layer is DW = sum_t g_t a_t^T, where a_t is the
 *     layer input and g_t the loss gradient w.r.t. the layer output at token t.
 *   - Sec. 3.2, Eq. (2) and App. A.2 "Factor projection": with maps
 *     P_a (k_in x d_in) and P_g (k_out x d_out), sum_t (P_a a_t) (x) (P_g g_t)
 *     = (P_a (x) P_g) vec(DW).  The library stores P_in = P_a^T and
 *     P_out = P_g^T and produces, per layer, the k_in x k_out block
 *         Psi[c][r] = sum_t (a_t . P_in[:,c]) (g_t . P_out[:,r])
 *     either in the FACTORED form (A P_in)^T (B P_out) or in the MATERIALIZED
 *     form (P_out^T (B^T A) P_in)^T; both are exact (Sec. 3.2, "FLOP-aware
 *     routing"; App. A.4 "Routing": routes are algebraically equivalent).
 *   - Sec. 3.2 "FLOP-aware routing" / App. A.4: the route is chosen per layer
 *     by a cost model; here the model is calibrated for MI355X.
 *   - GradDot scoring (Sec. 4.1; gradient similarity, Sec. 2) with an optional
 *     positive diagonal preconditioner: S = (Phi_q diag(d)) Phi_train^T, and
 *     per-query top-k.
 *   - Sec. 3.2 / App. A.2 / App. B: K-FAC and EK-FAC curvature fitted on the
 *     projected factors, and queries preconditioned with it before scoring.
 *
 * Conventions for every entry point
 *   - All functions are extern "C" and never throw or abort; each returns a
 *     dattri_status.  On failure a message is available from
 *     dattri_last_error() (thread-local, valid until the next call on the
 *     same thread) and no output buffer has been written.
 *   - Argument, shape, dtype, state and workspace checks all happen on the
 *     host before any GPU work is enqueued.
 *   - Every device buffer is owned by the caller.  The library never
 *     allocates device memory; it reports the sizes it needs.
 *   - GPU work is enqueued on the stream given (a hipStream_t passed as
 *     void*, NULL = the default stream) and is asynchronous: results are valid
 *     once that stream has reached the point after the call.  Faults inside a
 *     kernel surface at the next synchronizing HIP call.
 *   - A context is not thread-safe: use one per thread (or per stream).
 *   - Layouts are row-major and dense unless a leading dimension is given.
 *     "bf16" is IEEE bfloat16; conversions to bf16 round to nearest even.
 */
#ifndef DATTRI_H
#define DATTRI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct dattri_ctx dattri_ctx;

/* Enumerations are int-sized.  Compiled as C++ they get a fixed int32_t
 * underlying type, so that any integer a caller passes is a value of the type
 * (and is then rejected by the argument checks if it names no enumerator)
 * rather than undefined behaviour. */
#ifdef __cplusplus
#define DATTRI_ENUM enum : int32_t
#else
#define DATTRI_ENUM enum
#endif

typedef DATTRI_ENUM {
  DATTRI_OK = 0,
  DATTRI_E_INVALID_ARG = -1, /* null pointer, out-of-range value, bad enum */
  DATTRI_E_SHAPE = -2,       /* sizes inconsistent with registration/capture */
  DATTRI_E_DTYPE = -3,       /* dtype not supported for this call */
  DATTRI_E_STATE = -4,       /* call out of order (e.g. nothing captured) */
  DATTRI_E_WORKSPACE = -5,   /* workspace missing or smaller than required */
  DATTRI_E_HIP = -6,         /* a HIP runtime call failed (message has it) */
  DATTRI_E_UNSUPPORTED = -7  /* valid request outside this build's limits */
} dattri_status;

typedef DATTRI_ENUM { DATTRI_F32 = 0, DATTRI_BF16 = 1 } dattri_dtype;

typedef DATTRI_ENUM {
  DATTRI_ROUTE_AUTO = 0,        /* per-layer choice of the cost model */
  DATTRI_ROUTE_FACTORED = 1,    /* (A P_in)^T (B P_out), Eq. (2) left side */
  DATTRI_ROUTE_MATERIALIZED = 2, /* G = B^T A, then P_out^T G P_in */
  DATTRI_ROUTE_MASK = 3          /* reported for mask layers only (gathered entries) */
} dattri_route;

/* Kernel form of the factored route.  Both compute Eq. (2)'s left side with
 * float32 accumulation; they differ only in how work is spread over the GPU:
 *   FUSED  one kernel per work item (input group, example, token chunk)
 *          projects A and B and contracts the tokens in registers;
 *   SPLIT  stage 1 projects all n*T token rows slab by slab over d (many
 *          small work items), stage 2 sums the slabs and contracts each
 *          example's tokens in chunks; suited to captures with few examples
 *          or short sequences, where the fused kernel has little parallelism.
 * AUTO picks SPLIT when the fused kernel would have fewer than 1024 work
 * items, and for input groups whose maps are wider than 48 columns on both
 * sides (the fused kernel then holds too few token rows per wave to stream
 * at full rate); FUSED otherwise. */
typedef DATTRI_ENUM {
  DATTRI_FORM_AUTO = 0,
  DATTRI_FORM_FUSED = 1,
  DATTRI_FORM_SPLIT = 2
} dattri_factored_form;

/* ---------------------------------------------------------------- context */

/* Create a context.  `compute` is the element type of the captured factor
 * blocks A, B and of the projection maps (inputs are never converted);
 * `seed` is the global seed from which every layer's two projection maps are
 * derived (App. A.2: distinct seeds per side derived from a per-layer base
 * seed, fixed across all gradients that are compared).
 * Errors: INVALID_ARG (out == NULL), DTYPE (unknown compute type). */
dattri_status dattri_create(dattri_ctx** out, dattri_dtype compute, uint64_t seed);

/* Destroy a context (NULL is allowed).  Does not synchronize any stream. */
void dattri_destroy(dattri_ctx* ctx);

/* Message of the most recent call on this thread if it failed, "" otherwise. */
const char* dattri_last_error(void);

/* ------------------------------------------------------------ layers / maps */

/* Register a linear layer z = W a with W in R^{d_out x d_in} (Sec. 3.2) and
 * projection dimensions k_in (input side, k_a) and k_out (output side, k_g).
 * Layer ids are 0, 1, 2, ... in registration order, which is also the order of
 * the layer blocks inside phi.  Block l occupies columns
 * [offset_l, offset_l + k_in*k_out) with element (c, r) at offset_l + c*k_out + r
 * (the Kronecker order of Eq. (2)).
 * Errors: INVALID_ARG (ctx/layer_id NULL, any size < 1, d or k > 2^20). */
dattri_status dattri_register_layer(dattri_ctx* ctx, int32_t d_in, int32_t d_out,
                                    int32_t k_in, int32_t k_out, int32_t* layer_id);

/* Register a mask layer (App. A.2 "Random maps": a random mask keeps a fixed
 * random subset M of the entries of DW, gathered from the factors as
 * sum_t g_{t,r} a_{t,c}, |M| products per token, DW never formed).  The
 * layer's block in phi holds masks mask_id .. mask_id + mask_count - 1 of the
 * layer, mask_size entries each, back to back (one pass over the factors
 * serves them all); inside a mask, entry e is DW[r_e][c_e], ordered by
 * u = c * d_out + r (Eq. 1's column-stacked order).  The masks are drawn from
 * the layer's seed: with base = SM(seed) and s = SM(base ^ (2^63 | layer)),
 * draw i is ((x0 << 32) | x1) mod (d_out d_in) for
 * (x0..x3) = Philox4x32-10(counter (i lo, i hi, 0, 0), key (s lo, s hi));
 * repeats are dropped (first occurrence kept) and mask j is run j of
 * mask_size consecutive distinct draws, so the masks of a layer are disjoint
 * (AdamW-influence uses ten of 512 or 8192 entries, App. B).  Such a layer is
 * always projected by the gather kernel (route DATTRI_ROUTE_MASK, whatever
 * route is requested); its "maps" are the entry table (dattri_projection_bytes
 * gives its size in bytes_in, 12 bytes per entry plus 16 per group of 16384
 * entries, 0 in bytes_out; dattri_bind_projection uploads it into dev_P_in,
 * dev_P_out may be NULL, overrides are refused).  The table is the library's
 * own: the entries in the gather kernel's slot order with their positions in
 * mask order, and per group the part of each token row that it reads.
 * dattri_layer_dims reports k_in = 1, k_out = mask_size * mask_count.
 * Curvature calls reject mask layers.
 * Errors: INVALID_ARG (NULL pointers, sizes outside [1, 2^20], mask_size or
 * mask_count < 1, more than 2^24 entries, (mask_id + mask_count) * mask_size
 * above half of d_in * d_out). */
dattri_status dattri_register_mask_layer(dattri_ctx* ctx, int32_t d_in, int32_t d_out,
                                         int32_t mask_size, int32_t mask_id, int32_t mask_count,
                                         int32_t* layer_id);

/* Host copy of a mask layer's entries (rows r_e and cols c_e, int32
 * [mask_size * mask_count] each, in block order; either output may be NULL).
 * Host-only.
 * Errors: INVALID_ARG (bad layer, not a mask layer). */
dattri_status dattri_get_mask(const dattri_ctx* ctx, int32_t layer, int32_t* rows, int32_t* cols);

/* Number of registered layers. */
dattri_status dattri_num_layers(const dattri_ctx* ctx, int32_t* n);

/* Registered sizes of a layer (any output may be NULL). */
dattri_status dattri_layer_dims(const dattri_ctx* ctx, int32_t layer, int32_t* d_in, int32_t* d_out,
                                int32_t* k_in, int32_t* k_out);

/* Total feature dimension F = sum_l k_in,l * k_out,l, and a layer's offset. */
dattri_status dattri_feature_dim(const dattri_ctx* ctx, int64_t* F);
dattri_status dattri_layer_offset(const dattri_ctx* ctx, int32_t layer, int64_t* offset);

/* Device bytes the caller must provide for the layer's two projection maps.
 * The maps are stored in an internal fragment-major layout (16-byte lane
 * fragments, zero padded); read them back with dattri_get_projection. */
dattri_status dattri_projection_bytes(const dattri_ctx* ctx, int32_t layer,
                                      size_t* bytes_in, size_t* bytes_out);

/* Generate (or take) the layer's projection maps and upload them into the
 * caller-owned device buffers dev_P_in / dev_P_out (at least the sizes from
 * dattri_projection_bytes, 16-byte aligned).  The library keeps the pointers:
 * the buffers must stay valid and unmodified while the context uses them.
 *
 * Seeded maps (override == NULL): Gaussian entries N(0, 1/k) with k the map's
 * output dimension (App. A.2 "Random maps"), drawn as
 *   s = SM(SM(seed) ^ (2*layer + side)),  side 0 = P_in, 1 = P_out,
 *   (x0..x3) = Philox4x32-10(counter = (e lo, e hi, 0, 0), key = (s lo, s hi)),
 *   e = v*k + c for element (v, c) of the d x k map,
 *   u1 = (((x0<<32|x1) >> 11) + 1) 2^-53,  u2 = ((x2<<32|x3) >> 11) 2^-53,
 *   P[v][c] = sqrt(-2 ln u1) cos(2 pi u2) / sqrt(k)     (in double),
 * where SM(x) is one SplitMix64 output from state x; then rounded to float32
 * (RNE) and, for a bf16 context, to bf16 (RNE).
 * Override: host_P_in [d_in x k_in] / host_P_out [d_out x k_out] float32
 * row-major replace the seeded map of that side (rounded to the compute type).
 * The upload is complete when the call returns (it synchronizes `stream`).
 * Errors: INVALID_ARG (bad layer, NULL or misaligned device pointer), HIP. */
dattri_status dattri_bind_projection(dattri_ctx* ctx, int32_t layer, void* dev_P_in,
                                     void* dev_P_out, const float* host_P_in_override,
                                     const float* host_P_out_override, void* stream);

/* Kind of a layer's seeded maps (App. A.2 "Random maps"): Gaussian entries
 * N(0, 1/k) (the default, drawn as described above) or Rademacher entries
 * +-1/sqrt(k), k the map's output dimension, with the sign of element
 * e = v*k + c taken from bit 31 of the first output word x0 of the same
 * Philox4x32-10 counter and key (set: negative).  Both sides of the layer use
 * the kind.  Changing the kind of a bound layer unbinds it (bind again before
 * projecting); overrides given at binding are unaffected by the kind.
 * Errors: INVALID_ARG (bad layer, unknown kind, NULL kind). */
typedef DATTRI_ENUM { DATTRI_MAP_GAUSSIAN = 0, DATTRI_MAP_RADEMACHER = 1 } dattri_map_kind;
dattri_status dattri_set_map_kind(dattri_ctx* ctx, int32_t layer, dattri_map_kind kind);
dattri_status dattri_get_map_kind(const dattri_ctx* ctx, int32_t layer, dattri_map_kind* kind);

/* Host copy of the maps the layer uses, after rounding to the compute type:
 * the seeded maps (whether or not bound yet) or the overrides given at
 * binding; float32 row-major [d_in x k_in] and [d_out x k_out].  Either
 * output may be NULL.  Host-only (no GPU needed).
 * Errors: INVALID_ARG (bad layer). */
dattri_status dattri_get_projection(const dattri_ctx* ctx, int32_t layer, float* host_P_in,
                                    float* host_P_out);

/* --------------------------------------------------------------- capture */

/* Record one layer's factor blocks for a batch of n examples (App. A.5: the
 * layer input and the output gradient, as a backward hook records them).
 *   A: device [n, T, d_in]  (row t of example i is a_t), compute dtype
 *   B: device [n, T, d_out] (row t of example i is g_t), compute dtype
 *   dev_lengths: NULL (every example has T tokens) or device int32 [n]; only
 *     the first lengths[i] token rows of example i contribute (variable T_i,
 *     Eq. (4)); values are clamped to [0, T] on the device.
 * Pointers are borrowed, not copied: they must stay valid and unmodified
 * until the GPU work of every call that reads them has completed.  Layers
 * that pass the same A pointer (same d_in, n, T, lengths) share one read of A
 * in the factored route (e.g. q/k/v projections of one attention block).
 * Every registered layer must be captured with the same n before projecting.
 * Errors: INVALID_ARG (bad layer, NULL A/B with n*T > 0, n < 0, T < 0),
 * SHAPE (n*T*d beyond 2^31 elements per example block). */
dattri_status dattri_capture_layer(dattri_ctx* ctx, int32_t layer, const void* A, const void* B,
                                   int32_t n, int32_t T, const int32_t* dev_lengths);

/* Forget every capture (pointers are no longer referenced afterwards). */
dattri_status dattri_clear_captures(dattri_ctx* ctx);

/* ------------------------------------------------------------- projection */

/* Bytes of workspace dattri_project_per_example needs for the current
 * captures with the given route override.  Materialized layers stage their
 * weight gradients G (float32, d_out x d_in per example) in the workspace, a
 * bounded number of examples at a time; `bytes` is the size this build plans
 * for (any workspace at least this large works).
 * Errors: STATE (a registered layer not captured, or captures disagree on n). */
dattri_status dattri_workspace_bytes(const dattri_ctx* ctx, dattri_route route, size_t* bytes);

/* Set / read the context's factored-route kernel form (default AUTO).
 * Errors: INVALID_ARG (NULL ctx, unknown form). */
dattri_status dattri_set_factored_form(dattri_ctx* ctx, dattri_factored_form form);
dattri_status dattri_get_factored_form(const dattri_ctx* ctx, dattri_factored_form* form);

/* Projected per-example gradients of every registered layer, concatenated
 * (Eq. (2) per layer; blocks in registration order).
 *   phi: device [n, ld_phi] of phi_dtype (F32 or BF16), ld_phi >= F; row i is
 *        example i of the captures; columns >= F are not written.
 *   workspace: device, >= dattri_workspace_bytes(route) bytes, 256-byte aligned.
 *   route: AUTO (cost model per layer) or a route forced for every layer.
 * Accumulation is float32 throughout; a bf16 phi is rounded once at the end.
 * Errors: STATE (maps not bound, captures missing/inconsistent), SHAPE,
 * WORKSPACE, UNSUPPORTED (factored route forced on a layer with k_in > 128
 * or k_out > 64), HIP. */
dattri_status dattri_project_per_example(dattri_ctx* ctx, void* phi, dattri_dtype phi_dtype,
                                         int64_t ld_phi, void* workspace, size_t ws_bytes,
                                         dattri_route route, void* stream);

/* Launch tables kept on the device between calls (optional).  Every call that
 * launches the projection kernels first puts its launch tables (work items,
 * layer-group and reduction descriptors) on the device.  Without a plan
 * buffer they are copied into the head of the call's workspace on every call.
 * With one bound, each kind of table (projection; the curvature fit's row and
 * factor-sum tables; EK-FAC; token scores; cross-Gram) has a slot in it, and a
 * call whose table equals the one already in its slot (same captures, maps,
 * route, form, cost model and workspace address) issues no host-to-device
 * copy at all.  A table larger than the buffer takes the workspace path.
 *   dev_plan: device, 256-byte aligned, `bytes` long; NULL unbinds.  The
 *     library keeps the pointer: the buffer must stay valid and must not be
 *     written by anything else while bound.  Calls that use it must be
 *     ordered (one stream, or synchronized between streams), as for the
 *     workspace.
 * dattri_plan_bytes: bytes the projection's tables need for the current
 * captures and route (a buffer of this size, or several times it for the
 * other table kinds, suffices).
 * Errors: INVALID_ARG (NULL ctx / bytes, misaligned buffer, unknown route),
 * STATE (as dattri_workspace_bytes). */
dattri_status dattri_bind_plan_buffer(dattri_ctx* ctx, void* dev_plan, size_t bytes);
dattri_status dattri_plan_bytes(const dattri_ctx* ctx, dattri_route route, size_t* bytes);

/* Materialized representation (Eq. (1)): G_i = B_i^T A_i = sum_t g_t a_t^T for
 * captured examples [ex_begin, ex_begin + ex_count) of one layer, written as
 * float32 G_out [ex_count, d_out, d_in] (device).  Needs no workspace.
 * Errors: INVALID_ARG (bad layer or range, NULL G_out), STATE (not captured), HIP. */
dattri_status dattri_materialize_gradient(dattri_ctx* ctx, int32_t layer, int32_t ex_begin,
                                          int32_t ex_count, float* G_out, void* stream);

/* ------------------------------------------------------------- cost model */

/* MI355X time model of the two routes (Sec. 3.2 "FLOP-aware routing", App. A.4:
 * the cheaper exact route is taken per layer).  For one layer captured with n
 * examples, in microseconds:
 *   factored      = call_us + max(F_f / factored_tflops, B_f / factored_gbs)
 *                   + launches_f * launch_us
 * with the exact FLOP and byte counts of dattri_layer_costs times n, and
 * launches_f the number of kernels the factored route runs for this layer
 * alone: 2 in the fused form (projection + reduction), 3 to 5 in the split
 * form (stage 1 per map width, slab sum, contraction, reduction), as the
 * launch plan decides.  The materialized route has two implementations:
 *   - one pass (bf16 blocks with 16-byte aligned rows, k_in <= 128): each
 *     workgroup forms 128 rows of G over a token chunk, 128 columns at a
 *     time, and projects every tile from its accumulators, so G never goes
 *     to memory;
 *       materialized = call_us + max(W, B_f / gradient_gbs) + chunks_e * launch_us,
 *     chunks_e the launches of at most 65535 examples each (the small
 *     reduction of partial products behind each is charged no launch of its
 *     own: on MI355X the pair's fixed cost measures about one launch), and
 *     W the work of its launch shape: rounds of 256 occ workgroups (occ
 *     per CU: 2 when k_in <= 64, else 1) times occ times, per workgroup and
 *     128-column tile, tok_chunk / 32 token stages at 256 x 2 x 32 x 128 x
 *     128 FLOP per round plus one tile projection (G split into three bf16
 *     terms) at 256 x 3 x 2 x 128 x 128 x 16 x tiles(k_in) FLOP per round,
 *     plus once per workgroup the closing H^T P_out, also three bf16 terms,
 *     at 256 x 3 x 2 x 128 x 16 tiles(k_in) x 32 tiles32(k_out) FLOP per
 *     round, all bf16 MFMA at gradient_tflops (tiles(k_in) = 2, 4 or 8, the
 *     16-column tiles of the instance), plus round_us per round (load
 *     latencies and barriers, whatever the work); the token chunks and
 *     column ranges are the ones that minimise W;
 *   - otherwise (float32, unaligned rows, k_in > 128) G is staged in the
 *     workspace, chunks_m example chunks of at most 2 GiB of G each:
 *       materialized = call_us + max(F_g / gradient_tflops, B_g / gradient_gbs)
 *                      + max(F_p / gproject_tflops, B_p / gproject_gbs)
 *                      + 3 * chunks_m * launch_us
 *     with F_g, B_g the G = B^T A kernel (2T d_in d_out FLOP, factor blocks
 *     read and G written) and F_p, B_p the projection of G (the rest of the
 *     materialized FLOPs, G read).
 * call_us is paid by both routes and does not change a decision.  Ties go to
 * the factored route.  Rates are effective ones, fitted on MI355X; they may
 * not exceed the chip's published peaks (HBM 8000 GB/s, dense bf16 MFMA
 * 2500 TFLOP/s for the factored and gradient kernels, float32 MFMA
 * 157.3 TFLOP/s for gproject_tflops, the float32 kernels' rate). */
typedef struct {
  double factored_tflops;     /* factored kernels (fused or split) */
  double factored_gbs;
  double gradient_tflops;     /* G = B^T A */
  double gradient_gbs;
  double gproject_tflops;     /* float32 MFMA: staged P_out^T G P_in */
  double gproject_gbs;
  double launch_us;           /* per kernel launch */
  double call_us;             /* per call, either route */
  double round_us;            /* fixed time of one round of one-pass workgroups */
} dattri_cost_model;

/* Replace / read the context's cost model.
 * Errors: INVALID_ARG (NULL, a rate not finite or <= 0 or above its peak,
 * launch_us, call_us or round_us negative or not finite). */
dattri_status dattri_set_cost_model(dattri_ctx* ctx, const dattri_cost_model* model);
dattri_status dattri_get_cost_model(const dattri_ctx* ctx, dattri_cost_model* model);

/* Load the cost model from a calibration file: a JSON object whose member
 * "model" is an object holding the nine fields of dattri_cost_model by name
 * as numbers (the file `python -m paper_2609_38767_amd.calibrate --out FILE`
 * writes; other members are ignored).  Host-only; reads the file once.  The
 * context's model is unchanged on error.
 * Errors: INVALID_ARG (NULL arguments, unreadable file, malformed JSON, no
 * "model" object, a field missing or not a number, a value rejected as by
 * dattri_set_cost_model). */
dattri_status dattri_set_cost_calibration(dattri_ctx* ctx, const char* json_path);

/* Exact per-example operation counts of a layer's two routes for T tokens
 * (any of the outputs may be NULL):
 *   factored FLOP      2T(d_in k_in + d_out k_out + k_in k_out)
 *   materialized FLOP  2T d_in d_out + 2 d_out d_in k_in + 2 d_out k_in k_out
 *                      (the association (G P_in) first, which this build runs)
 *   factored bytes     T (d_in + d_out) elt      (factor blocks read once)
 *   materialized bytes factored bytes + 2 * 4 d_out d_in (G written and read;
 *                      the one-pass kernel keeps G on chip and reads only the
 *                      factored bytes)
 * Errors: INVALID_ARG (bad layer, T < 0). */
dattri_status dattri_layer_costs(const dattri_ctx* ctx, int32_t layer, int32_t T,
                                 int64_t* factored_flops, int64_t* materialized_flops,
                                 int64_t* factored_bytes, int64_t* materialized_bytes);

/* Route an AUTO call over the context's captured layers takes for a layer,
 * with both predicted times of the layer alone in microseconds.  Each layer
 * is first decided on its own (ties go to FACTORED).  Then, when some layer of
 * the call is factored, the factored launches are paid and shared anyway, so a
 * layer decided MATERIALIZED joins the factored route if its predicted
 * factored time without launch costs is no more than its materialized time
 * (each materialized layer adds launches of its own).  A layer whose k
 * exceeds the factored kernel's limits (k_in > 128 or k_out > 64) always
 * routes MATERIALIZED (its predicted factored time is infinite).
 * Errors: INVALID_ARG (bad layer), STATE (layer not captured). */
dattri_status dattri_layer_route(const dattri_ctx* ctx, int32_t layer, dattri_route* chosen,
                                 double* pred_factored_us, double* pred_materialized_us);

/* ------------------------------------------- unprojected cross-Gram matrices */

/* Sec. 3.2 "Factorized inner product" (Eq. 4) and "FLOP-aware routing"; App.
 * A.4 (routing-complexity table, "Routing").  For the captures of two contexts
 * a (n_a examples) and b (n_b examples) over the same registered layers, the
 * cross-Gram matrix of their unprojected per-example weight gradients summed
 * over layers:
 *     K[i][j] = sum_l < DW_l^(a,i), DW_l^(b,j) >_F
 * Per layer one of two exact routes computes the contribution:
 *   FACTORED      Eq. 4: sum over token pairs (t < T_i, s < T_j) of
 *                 <a_t, a_s> <g_t, g_s>, i.e. the entries of
 *                 (A_i A_j^T) * (B_i B_j^T) summed; cost ~ n_a n_b T^2 (d_in + d_out);
 *   MATERIALIZED  DW = B^T A for every example (Eq. 1), then Frobenius
 *                 products; cost ~ (n_a + n_b) T d_in d_out + n_a n_b d_in d_out.
 * The projection sizes k_in / k_out and the maps play no part here.  The two
 * contexts must have the same compute type and the same layer list (count,
 * d_in, d_out); a and b may be the same context (the Gram of one batch).
 * Every layer must be captured in both; lengths apply as in projection. */

/* Rates of the cross-Gram time model (MI355X-fitted defaults).  Predicted time
 * of a layer's route:
 *   factored      max(tile_flops / ghost rate, tile_bytes / ghost bandwidth)
 *                 + ghost_layer_us, where the kernel computes whole 128 x 128
 *                 tiles of the token Gram (token rows padded to multiples of
 *                 16): tile_flops = tiles * 2 * 128^2 (d_in + d_out + 1),
 *                 tile_bytes = tiles * 2 * 128 (d_in + d_out) elt;
 *   materialized  the faster of two forms of Eq. 1 + Frobenius products:
 *                 staged: max(build rounds, build_bytes / build bandwidth)
 *                 + dot_bytes / dot bandwidth + 4 launch_us (DW of both
 *                 batches written to the workspace, then the products), where
 *                 the build runs one workgroup per 128 x 128 tile of DW and
 *                 example, per batch ceil(tiles n / 512) rounds of one tile
 *                 build, 2 * 128^2 * T (T rounded up to 32) FLOP at
 *                 build_tflops / 512;
 *                 one-pass (bf16 blocks with 16-byte aligned rows only): no DW
 *                 in memory, a workgroup forms one 128 x 128 tile of DW_b[j]
 *                 and then the same tile of DW_a[i] for each of a run of
 *                 ipw <= 4 examples, summing their products (all one-pass
 *                 layers of a call share one launch); predicted per layer as
 *                 rounds of 512 workgroups, each round ipw + 1 tile builds of
 *                 2 * 128^2 * T (T rounded up to 32) FLOP at onepass_tflops / 512,
 *                 plus 2 launch_us,
 * with build and product counts as in dattri_cross_gram_costs.  For the squared
 * norms the factorized tiles cover each example's own token Gram, the staged
 * products read DW once (3 launches), and the one-pass form has no reference
 * build. */
typedef struct {
  double ghost_tflops;   /* factorized kernel (two token Grams and their product) */
  double ghost_gbs;      /* its factor-block reads */
  double ghost_layer_us; /* fixed cost per layer inside the grouped factorized launch */
  double build_tflops;   /* DW = B^T A kernel */
  double build_gbs;      /* its factor reads plus float32 DW writes */
  double dot_gbs;        /* Frobenius products over stored float32 DW */
  double launch_us;      /* per kernel launch (staged materialized: four per layer) */
  double onepass_tflops; /* one-pass materialized kernel, on the tile builds it issues */
} dattri_crossgram_cost_model;

dattri_status dattri_set_crossgram_cost_model(dattri_ctx* ctx, const dattri_crossgram_cost_model* m);
dattri_status dattri_get_crossgram_cost_model(const dattri_ctx* ctx, dattri_crossgram_cost_model* m);

/* Exact operation counts of one layer's cross-Gram contribution between n_a
 * examples of T_a tokens and n_b examples of T_b tokens (any output may be
 * NULL); multiply-add = 2 FLOP:
 *   factored FLOP      2 n_a n_b T_a T_b (d_in + d_out + 1)
 *   materialized FLOP  2 (n_a T_a + n_b T_b) d_in d_out + 2 n_a n_b d_in d_out
 *   factored bytes     (n_a T_a + n_b T_b)(d_in + d_out) elt   (factor blocks)
 *   materialized bytes factored bytes + 2 * 4 (n_a + n_b) d_in d_out
 * Errors: INVALID_ARG (negative sizes, elt not 2 or 4). */
dattri_status dattri_cross_gram_costs(int64_t n_a, int64_t n_b, int32_t T_a, int32_t T_b,
                                      int32_t d_in, int32_t d_out, int32_t elt_bytes,
                                      int64_t* factored_flops, int64_t* materialized_flops,
                                      int64_t* factored_bytes, int64_t* materialized_bytes);

/* Route the cost model (of context a) picks for one layer's cross-Gram
 * contribution given the current captures, with both predicted times in
 * microseconds (ties go to FACTORED).
 * Errors: INVALID_ARG (bad layer), STATE (not captured), SHAPE (layer lists
 * or dtypes differ). */
dattri_status dattri_cross_gram_route(const dattri_ctx* a, const dattri_ctx* b, int32_t layer,
                                      dattri_route* chosen, double* pred_factored_us,
                                      double* pred_materialized_us);

/* Device bytes of workspace dattri_cross_gram needs for the current captures
 * and route (AUTO: the per-layer choice).  b == a is allowed.
 * Errors: as dattri_cross_gram_route. */
dattri_status dattri_cross_gram_workspace_bytes(const dattri_ctx* a, const dattri_ctx* b,
                                                dattri_route route, size_t* bytes);

/* K = cross-Gram of the captures of a (rows) and b (columns), as above.
 *   K: device float32 [n_a rows of ld_k >= n_b]; every element (i < n_a,
 *      j < n_b) is written, the rest of each row is not.
 *   workspace: device, >= dattri_cross_gram_workspace_bytes(a, b, route),
 *      256-byte aligned.
 *   route: AUTO (per layer by the cost model) or forced for every layer.
 * Accumulation is float32 (inputs in their own type, float32 products); the
 * result is deterministic (fixed summation order, no atomics).
 * Errors: INVALID_ARG, STATE, SHAPE, WORKSPACE, HIP. */
dattri_status dattri_cross_gram(dattri_ctx* a, dattri_ctx* b, float* K, int64_t ld_k,
                                void* workspace, size_t ws_bytes, dattri_route route,
                                void* stream);

/* Per-example squared gradient norms of one context's captures summed over
 * layers: out[i] = sum_l ||DW_l^(i)||_F^2 (the diagonal of the batch's Gram,
 * App. A.4 "Routing": norms are routed like cross-Grams; the factored route
 * costs 2 n T^2 (d_in + d_out + 1) per layer, the materialized one
 * 2 n T d_in d_out + 2 n d_in d_out).
 *   out: device float32 [n].
 *   workspace: >= dattri_sq_norms_workspace_bytes(ctx, route).
 * Errors: as dattri_cross_gram. */
dattri_status dattri_sq_norms_workspace_bytes(const dattri_ctx* ctx, dattri_route route,
                                              size_t* bytes);
dattri_status dattri_gradient_sq_norms(dattri_ctx* ctx, float* out, void* workspace,
                                       size_t ws_bytes, dattri_route route, void* stream);

/* ---------------------------------------------------------------- scoring */

/* Workspace bytes dattri_score needs for these sizes.  `has_precond` and
 * `has_scores` say whether dev_precond_diag and scores will be non-NULL. */
dattri_status dattri_score_workspace_bytes(int64_t n_q, int64_t n_train, int64_t F,
                                           dattri_dtype dtype, int32_t has_precond,
                                           int32_t has_scores, int32_t topk, size_t* bytes);

/* Recommended row stride (elements) for storing feature rows of F elements
 * of `dtype` (phi from dattri_project_per_example, or any phi_q / phi_train
 * given to dattri_score): F rounded up to 256 bytes, plus 512 bytes when the
 * row would otherwise be a multiple of 8 KiB of at least 16 KiB.  Such strides
 * map one column of many rows into the same few L2 sets of MI355X, and the
 * score GEMM then re-fetches operands it should share from memory.  Any
 * stride >= F is accepted by dattri_score; this one runs fastest.
 * Errors: INVALID_ARG (ld NULL, F < 0), DTYPE. */
dattri_status dattri_feature_ld(int64_t F, dattri_dtype dtype, int64_t* ld);

/* GradDot scores with an optional diagonal preconditioner, and top-k.
 *   phi_q:     device [n_q rows of F] of dtype, rows ld_q elements apart
 *   phi_train: device [n_train rows of F] of dtype, rows ld_train apart
 *   ld_q, ld_train: row strides in elements (0 = F, dense); >= F, and
 *              ld * element size a multiple of 16 bytes
 *   dev_precond_diag: NULL (d = 1) or device float32 [F], d > 0, applied once:
 *              S[q][j] = sum_f phi_q[q][f] d[f] phi_train[j][f].  For bf16 the
 *              query row is scaled in float32 and rounded once to bf16 (into
 *              the workspace, rows dattri_feature_ld apart).
 *   scores:    device float32 [n_q, n_train], or NULL if only top-k is wanted
 *   topk:      0 (no selection) or 1 <= topk <= min(n_train, 1024)
 *   topk_idx:  device int32 [n_q, topk]; topk_val: device float32 [n_q, topk]:
 *              per query the topk largest scores, largest first; equal scores
 *              are ordered by lower training index (-0.0 equals +0.0; NaN
 *              scores are not supported).
 *   workspace: device, >= dattri_score_workspace_bytes(...), 256-byte aligned.
 * Accumulation is float32.  Errors: INVALID_ARG (including ld < F), DTYPE,
 * WORKSPACE, UNSUPPORTED (topk > 1024, misaligned rows, 256 rows of the
 * stride reaching 4 GiB), HIP. */
dattri_status dattri_score(const void* phi_q, int64_t n_q, int64_t ld_q, const void* phi_train,
                           int64_t n_train, int64_t ld_train, int64_t F, dattri_dtype dtype,
                           const float* dev_precond_diag, float* scores, int32_t topk,
                           int32_t* topk_idx, float* topk_val, void* workspace, size_t ws_bytes,
                           void* stream);

/* Scoring for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation.  The
 * arguments, checks and results are those of dattri_score without the
 * workspace: its scratch (prepared queries, split-feature partial tiles, and
 * the scores themselves when `scores` is NULL and only top-k is wanted) lives
 * in a static device array of DATTRI_NOALLOC_SCRATCH_BYTES that the library
 * holds on every GPU it runs on until the process ends.  The call allocates
 * nothing.  Nothing in the scratch needs to start at zero: each call writes
 * every byte of it that it reads.  All calls on one GPU share its array and
 * the next call overwrites it: calls that overlap in time on one GPU (other
 * streams, other threads) race, and the caller must order them.
 * Errors: as dattri_score, plus UNSUPPORTED when the call would need more
 * scratch than DATTRI_NOALLOC_SCRATCH_BYTES (the 2048 x 8192 bf16 queries of
 * the scoring workload take 33.5 MB; top-k alone over 2048 x 200000 scores
 * needs 1.6 GB and is refused). */
#define DATTRI_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
dattri_status dattri_score_noalloc(const void* phi_q, int64_t n_q, int64_t ld_q, const void* phi_train,
                                   int64_t n_train, int64_t ld_train, int64_t F, dattri_dtype dtype,
                                   const float* dev_precond_diag, float* scores, int32_t topk,
                                   int32_t* topk_idx, float* topk_val, void* stream);

/* Cosine scores (Grad-Cos, Sec. 2; LESS's cosine metric, App. A.3): the same
 * call as dattri_score, with every score divided by the norms of its two rows,
 *   S[q][j] = <q', x_j> / (|q'| |x_j|),  q' = phi_q[q] * d (d = 1 when NULL),
 * and 0 when either norm is 0; top-k ranks these cosines.  Norms are float32
 * sums of squares of the rows as given (the query scaled by d in float32).
 *   workspace: >= dattri_cosine_workspace_bytes(...) (dattri_score's plus
 *   n_q + n_train floats), 256-byte aligned.
 * Errors: as dattri_score. */
dattri_status dattri_cosine_workspace_bytes(int64_t n_q, int64_t n_train, int64_t F,
                                            dattri_dtype dtype, int32_t has_precond,
                                            int32_t has_scores, int32_t topk, size_t* bytes);
dattri_status dattri_score_cosine(const void* phi_q, int64_t n_q, int64_t ld_q,
                                  const void* phi_train, int64_t n_train, int64_t ld_train,
                                  int64_t F, dattri_dtype dtype, const float* dev_precond_diag,
                                  float* scores, int32_t topk, int32_t* topk_idx, float* topk_val,
                                  void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------ K-FAC / EK-FAC curvature */

/* Kronecker-factored curvature on projected factors.  Sec. 3.2 names the
 * preconditioned comparisons of K-FAC (Martens & Grosse, 2015) and EK-FAC
 * (George et al., 2018) among the operations on factorized gradients, and
 * App. A.2 ("Factor projection") applies them unchanged to the projected
 * pair a~_t = P_in^T a_t, g~_t = P_out^T g_t.  Per layer:
 *
 *   input factor     A = (1/N_tok) sum over examples and tokens of a~ a~^T
 *   gradient factor  S = (1/N)     sum over examples and tokens of g~ g~^T
 *   eigenbases       A = Q_A diag(lam_A) Q_A^T,  S = Q_G diag(lam_G) Q_G^T
 *   eigenvalues      K-FAC   E[c][r] = lam_A[c] lam_G[r]
 *                    EK-FAC  E[c][r] = (1/N) sum_i ((Q_A^T Psi_i Q_G)[c][r])^2
 *   damping          delta = rel * mean(E) + abs   (App. B: rel = 0.1)
 *   preconditioned   P(Psi_q) = Q_A [(Q_A^T Psi_q Q_G) / (E + delta)] Q_G^T
 *
 * with Psi the layer's k_in x k_out block of phi (Eq. (2)), N_tok the token
 * positions and N the examples summed.  Scores of preconditioned queries
 * against training features come from dattri_score with no diagonal: the sum
 * over layers of <P(Psi_q), Psi_j>_F.
 *
 * All statistics live in one caller-owned device buffer, the curvature state
 * (dattri_curvature_state_bytes, 256-byte aligned).  Its per-layer fields are
 * at the byte offsets of dattri_curvature_layout_of; matrices are float32
 * row-major.  Sums accumulate over calls until dattri_curvature_reset.
 * Layers need k_in <= 64 and k_out <= 64 (else UNSUPPORTED). */
typedef DATTRI_ENUM { DATTRI_CURV_KFAC = 0, DATTRI_CURV_EKFAC = 1 } dattri_curvature;

typedef struct {
  int64_t sum_a;   /* float32 [k_in][k_in]:  sum of a~ a~^T                         */
  int64_t sum_g;   /* float32 [k_out][k_out]: sum of g~ g~^T                        */
  int64_t sum_e;   /* float32 [k_in][k_out]: sum over examples of (Q_A^T Psi Q_G)^2 */
  int64_t q_a;     /* float32 [k_in][k_in]: column j = eigenvector of lam_a[j]      */
  int64_t lam_a;   /* float32 [k_in], ascending                                     */
  int64_t q_g;     /* float32 [k_out][k_out]                                        */
  int64_t lam_g;   /* float32 [k_out], ascending                                    */
  int64_t counts;  /* int64 [3]: N_tok of sum_a, N of sum_g, N of sum_e             */
} dattri_curvature_layout;

/* Bytes of the curvature state of every registered layer.
 * Errors: INVALID_ARG, UNSUPPORTED (a layer with k_in or k_out > 64). */
dattri_status dattri_curvature_state_bytes(const dattri_ctx* ctx, size_t* bytes);
dattri_status dattri_curvature_layout_of(const dattri_ctx* ctx, int32_t layer,
                                         dattri_curvature_layout* out);

/* Zero every sum and count of a state (a fill kernel; no memset node). */
dattri_status dattri_curvature_reset(const dattri_ctx* ctx, void* state, void* stream);

/* Adds the projected factor sums of the current captures of every layer
 * (sum_a, sum_g and their counts; token rows past lengths[i] are left out).
 * One pass over A and B per layer side, each token row projected with the
 * layer's maps and its outer product accumulated in float32; the order of
 * every sum is fixed (deterministic, no atomics).
 *   workspace: >= dattri_curvature_fit_workspace_bytes(ctx), 256-byte aligned.
 * Errors: INVALID_ARG, STATE (maps not bound, captures missing or
 * inconsistent), WORKSPACE, UNSUPPORTED, HIP. */
dattri_status dattri_curvature_fit_workspace_bytes(const dattri_ctx* ctx, size_t* bytes);
dattri_status dattri_curvature_accumulate_factors(dattri_ctx* ctx, void* state, void* workspace,
                                                  size_t ws_bytes, void* stream);

/* Projected per-example gradients (exactly as dattri_project_per_example)
 * and the projected factor sums of the same captures (as
 * dattri_curvature_accumulate_factors), in one pass over A and B: the
 * factored kernels also keep each layer's projected token rows a~_t, g~_t
 * (float32, in the workspace) and the sums are formed from those rows; layers
 * on the materialized route, which never form projected rows, take the
 * separate factor-sum pass.
 *   workspace: >= dattri_project_fit_workspace_bytes(ctx, route), 256-byte aligned.
 * Errors: those of dattri_project_per_example and of
 * dattri_curvature_accumulate_factors. */
dattri_status dattri_project_fit_workspace_bytes(const dattri_ctx* ctx, dattri_route route,
                                                 size_t* bytes);
dattri_status dattri_project_and_fit(dattri_ctx* ctx, void* phi, dattri_dtype phi_dtype,
                                     int64_t ld_phi, void* state, void* workspace, size_t ws_bytes,
                                     dattri_route route, void* stream);

/* Eigendecomposition of every layer's normalized factors A and S (cyclic
 * parallel Jacobi in float64 on the GPU, one workgroup per factor, until the
 * off-diagonal mass falls below 1e-26 of the total or 32 sweeps); writes q_a,
 * lam_a, q_g, lam_g.  A factor with a zero count yields zeros and Q = I.
 * Errors: INVALID_ARG, UNSUPPORTED, HIP. */
dattri_status dattri_curvature_eigen(const dattri_ctx* ctx, void* state, void* stream);

/* EK-FAC's eigenvalue correction: adds, for every layer, the squared blocks
 * of n training rows of phi rotated into the layer's eigenbasis (needs
 * dattri_curvature_eigen first) to sum_e, and n to its count.
 *   phi: device [n rows of F] of dtype (F32 or BF16), rows ld elements apart
 *        (ld >= F).
 *   workspace: >= dattri_curvature_ekfac_workspace_bytes(ctx, n), 256-byte aligned.
 * Errors: INVALID_ARG, DTYPE, SHAPE, WORKSPACE, UNSUPPORTED, HIP. */
dattri_status dattri_curvature_ekfac_workspace_bytes(const dattri_ctx* ctx, int64_t n,
                                                     size_t* bytes);
dattri_status dattri_curvature_accumulate_ekfac(const dattri_ctx* ctx, void* state,
                                                const void* phi, dattri_dtype dtype, int64_t n,
                                                int64_t ld, void* workspace, size_t ws_bytes,
                                                void* stream);

/* Preconditioned query features: every layer block of n_q rows of phi_q
 * replaced by P(Psi_q) for curvature `kind` with damping
 * delta = damping_rel * mean(E) + damping_abs, computed in float32 and
 * written as out_dtype (bf16 rounded once).  EK-FAC needs
 * dattri_curvature_accumulate_ekfac first (with no correction its eigenvalues
 * read as zero); both kinds need dattri_curvature_eigen.
 *   phi_q: device [n_q rows of F] of in_dtype, rows ld_q apart (>= F)
 *   out:   device [n_q rows of F] of out_dtype, rows ld_out apart (>= F);
 *          columns >= F are not written; out must not overlap phi_q.
 * Errors: INVALID_ARG (damping_rel < 0, damping_abs < 0 or both zero),
 * DTYPE, SHAPE, UNSUPPORTED, HIP. */
dattri_status dattri_curvature_precondition(const dattri_ctx* ctx, const void* state,
                                            dattri_curvature kind, double damping_rel,
                                            double damping_abs, const void* phi_q,
                                            dattri_dtype in_dtype, int64_t n_q, int64_t ld_q,
                                            void* out, dattri_dtype out_dtype, int64_t ld_out,
                                            void* stream);

/* ------------------------------------------------- token-level attribution */

/* Token-level scores (App. D: the contribution of token t of training example
 * i to its score against query j is g_t^T R^(j) a_t, and the contributions sum
 * to <DW^(i), R^(j)>_F; summed over layers).  On projected factors the
 * layer's query-side matrix is the query row's k_in x k_out block R (element
 * (c, r) the coefficient of a~_t[c] g~_t[r], the layout of phi), so
 *   scores[q][i][t] = sum over layers of a~_t^T R_q g~_t,
 * and sum_t scores[q][i][t] = <phi_q[q], phi[i]> (GradDot for the query's own
 * phi row; K-FAC / EK-FAC for rows from dattri_curvature_precondition).
 * Positions at or past a layer's length for example i add nothing.
 * The call also projects the current captures (every layer on the factored
 * route, which forms the projected rows) and writes their phi when `phi` is
 * given (as dattri_project_per_example; NULL keeps it in the workspace).
 *   phi_q:  device [n_q rows of F] of q_dtype, rows ld_q apart (>= F)
 *   scores: device float32 [n_q][n][T]
 *   workspace: >= dattri_token_scores_workspace_bytes(ctx), 256-byte aligned.
 * Layers need k_in, k_out <= 64, one T for all captures, no mask layers.
 * Errors: INVALID_ARG, DTYPE, SHAPE, STATE, WORKSPACE, UNSUPPORTED, HIP. */
dattri_status dattri_token_scores_workspace_bytes(const dattri_ctx* ctx, size_t* bytes);
dattri_status dattri_token_scores(dattri_ctx* ctx, const void* phi_q, dattri_dtype q_dtype,
                                  int64_t n_q, int64_t ld_q, float* scores, void* phi,
                                  dattri_dtype phi_dtype, int64_t ld_phi, void* workspace,
                                  size_t ws_bytes, void* stream);

/* ------------------------------------------------------ measurement probes */

/* Measured roofline denominators (not part of the method): the rates a kernel
 * of this library is also compared against, besides the published peaks.
 *
 * dattri_probe_read: one launch of `workgroups` x 256 threads that reads
 * `bytes` of device memory at buf once (non-temporal 16-byte loads,
 * grid-stride) and writes one int32 per thread to sink; time it on `stream`
 * to get the achievable HBM read rate.
 *   buf:  device, 16-byte aligned; bytes a positive multiple of 16
 *   sink: device int32 [workgroups * 256] (caller-owned, contents unspecified)
 * Errors: INVALID_ARG, HIP.
 *
 * dattri_probe_mfma: one launch of `workgroups` x 4 waves, each issuing
 * iters x 8 independent bf16 MFMA 32x32x16 operations from registers (no
 * memory traffic in the loop); *flops receives the launch's FLOP count
 * (workgroups x 4 x iters x 8 x 32768).  Time it on `stream` to get the
 * achievable dense bf16 matrix rate, clock throttling included.
 *   sink: device float32 [workgroups * 256] (caller-owned, contents unspecified)
 * Errors: INVALID_ARG (iters < 1, workgroups outside [1, 2^20]), HIP. */
dattri_status dattri_probe_read(const void* buf, size_t bytes, int32_t* sink, int32_t workgroups,
                                void* stream);
dattri_status dattri_probe_mfma(float* sink, int32_t workgroups, int32_t iters, double* flops,
                                void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DATTRI_H */
