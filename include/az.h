/*
 * az.h - C ABI of the MI355X (gfx950) library that evaluates the residual
 * policy/value network on batches of search-leaf positions.
 *
 * What it computes.  In the paper's self-play loop every new search leaf that
 * is not terminal is sent to the network; requests from many games are grouped
 * into one batch and evaluated on the GPU, which returns move priors over the
 * legal moves and a scalar value (Section 3.3 "One learning cycle", Section 3.6
 * "Search and self-play", Section 5.2 "Batching and host-side submission").
 * For each position b of a batch this library computes
 *
 *   h      = act(conv3x3(planes[b]) + b_stem)                 stem ("start block")
 *   t      = act(conv3x3(h) + b1_j)                           block j = 0..blocks-1
 *   h      = act(h + conv3x3(t) + b2_j)                       (post-activation residual block)
 *   z[i]   = b_p[p] + sum_f Wp[p][f] * h[f][r][c],  i = p*64 + r*8 + c   (move-plane head)
 *   P[i]   = exp(z[i] - m) / sum_{k legal} exp(z[k] - m) if legal[b][i] != 0, else 0,
 *            m = max over legal z; a row with no legal cell is all zero
 *   u[s]   = b_v + sum_f w_v[f] * h[f][s]   (then ReLU if value_conv_relu)
 *   V      = tanh(w2 . relu(W1 u + b1) + b2)
 *
 * conv3x3 is a stride-1 3x3 cross-correlation with a zero pad of one square on
 * each 8x8 board; act is ReLU, capped at act_cap when act_cap > 0 (the capped
 * activation of Section 4.3, "Quantization as an architectural constraint").
 * Batch normalisation and any residual-branch scale are folded into the
 * weights by the caller, as the paper does on its deployment copy (Section 4.3,
 * Appendix D).
 *
 * Precision (Section 5.3 "Inference runtimes and precision": most trunk
 * convolutions in INT8, start block, heads and linear layers at higher
 * precision):
 *   AZ_F32       every layer in fp32.
 *   AZ_BF16      bf16 weights and activations, fp32 accumulation; heads fp32
 *                accumulation, softmax and value in fp32.
 *   AZ_INT8      the 2*blocks residual convolutions in int8 with exact int32
 *                accumulation: weights quantised per output channel
 *                (q = sat(rne(w / s_w[f])), |q| <= 127, the quotient decided
 *                exactly), every activation tensor between layers stored as
 *                int8 codes with a per-tensor scale.  The stem runs in bf16 and
 *                quantises its output; heads, softmax and value in fp32.
 *   AZ_FP8_E4M3  as AZ_INT8 with OCP fp8 e4m3 codes (max 448, saturating,
 *                round to nearest even).  The definition sums e4m3 products
 *                exactly; the gfx950 e4m3 matrix instruction does not: it sums
 *                runs of 8 consecutive input channels of one tap with every
 *                product truncated toward zero to 2^(E-13), E the largest
 *                exponent among that run's nonzero products, and adds each run's
 *                sum to an fp32 accumulator.  On deep networks the results
 *                therefore drift from the definition (a 20-block, 128-filter
 *                network: max |dP| about 0.09, |dV| about 0.5); AZ_INT8 is the
 *                format that computes the definition.
 *   Heads (1x1 policy and value convolutions) use bf16-rounded weights with fp32
 *   accumulation under every dtype except AZ_F32.
 *   For AZ_INT8 / AZ_FP8_E4M3 the codes are defined by (a[k] the activation
 *   scale of tensor k: the stem writes tensor 0, residual conv n = 2j (first
 *   of block j) or 2j+1 (second) writes tensor k = n+1):
 *           y = acc * a[n] * s_w[n][f] + b[f]       (acc: sum of code products)
 *           (second conv only) y += q_res * a[k-2]  (q_res: the block input's code)
 *           q = sat(rne(act(y) / a[k]))
 *   and the stem writes q = sat(rne(act(acc + b[f]) / a[0])) from its bf16
 *   sums; the heads take q * a[2*blocks].  The library evaluates z = act(y) /
 *   a[k] in float64, as z = acc * (a[n] s_w[n][f] / a[k]) + b[f] / a[k]
 *   (+ q_res * a[k-2] / a[k]) clamped to [0, min(qmax, act_cap / a[k])], so a
 *   code can differ from exact arithmetic only within about 2^-45 of a
 *   rounding tie.  The stem's sums come from the bf16 matrix instruction in
 *   fp32 (exact while every partial sum is an fp32 value).
 *
 * The deployed network (Section 3.5 "Chess representation and outputs",
 * Section 4.3 "Convolution, attention, and global context", "Three policy
 * representations", "Value and training-only heads", Appendix D) is selected by
 * the version-2 spec fields and changes three things:
 *   global pooling   (pool_every = p > 0) blocks j with j % p == p - 1 split
 *                    their first convolution's F outputs into Fr = F - F/4
 *                    regular and g = F/4 pooled channels (the last g):
 *                      z  = conv3x3(h) + b1
 *                      pc = act(z[Fr + i]),  i < g
 *                      gv = [mean over squares of pc_i (i < g), max over squares of pc_i (i < g)]
 *                      c  = Wg gv                         (Wg is [Fr][2g])
 *                      t  = act(z[0:Fr] + c)
 *                      h  = act(h + conv3x3(t) + b2)      (W2 is [F][Fr][3][3])
 *   from-to policy   (policy_head = AZ_POLICY_FROMTO, token_dim D)
 *                      tok[s] = relu(We h[:, s] + be),  Q[s] = Wq tok[s] + bq,
 *                      K[s] = Wk tok[s] + bk,  S[f][t] = Q[f] . K[t] / sqrt(D),
 *                      O[c][k] = Wp[k] . K[56 + c]
 *                    over 1,880 actions: the 1,792 origin-destination pairs f -> t
 *                    on a common row, column or diagonal or a knight's jump apart,
 *                    ascending (f, t), logit S[f][t]; then the 88 promotions, f on
 *                    row 6, t on row 7 at most one column away, piece k = 0..3
 *                    (queen, rook, bishop, knight), ascending (f, t, k), logit
 *                    S[f][t] + O[t - 56][k].  Squares are row * 8 + column in
 *                    the side-to-move frame.  The legal-action softmax is the
 *                    one above, over these 1,880 logits.
 *   WDL value        (value_head = AZ_VALUE_WDL, value_channels V)
 *                      u = Wv h + bv (V x 64, then ReLU if value_conv_relu),
 *                      y = relu(W1 u + b1) (u flattened channel-major),
 *                      (W, D, L) = softmax(W2 y + b2),  value = W - L.
 * In AZ_INT8 the pooled channels' mean, maximum and projection are taken in
 * floating point inside the integer trunk: pc = act(acc * a[n] * s_w[n][f] +
 * b1[f]) from the exact integer sums, the statistics and c = Wg gv in float64,
 * and c joins the regular channels' y before their activation and rounding
 * (all in float64); the pooled channels are stored as codes like any other
 * output and read by nothing.  Heads run on bf16 operands with split (hi + lo)
 * products and fp32 accumulation, softmax and WDL in fp32.
 *
 * Threading and streams.  Evaluation only reads a handle (it keeps no
 * workspace), so az_eval_batch may run concurrently on one handle from several
 * threads and streams; az_net_set_tiling and az_net_free must not run
 * concurrently with evaluations on the same handle.  A pipeline (below) is used
 * by one thread at a time.  az_last_error() is thread-local.
 */
#ifndef AZ_H
#define AZ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define AZ_ABI_VERSION 2
#define AZ_SQUARES 64

typedef struct az_net az_net; /* opaque: owns the device copy of the packed weights */

typedef enum {
  AZ_F32 = 0,
  AZ_BF16 = 1,
  AZ_INT8 = 2,
  AZ_FP8_E4M3 = 3
} az_dtype;

typedef enum {
  AZ_OK = 0,
  AZ_ERR_INVALID_ARG = -1, /* NULL pointer, bad size or count, misaligned buffer */
  AZ_ERR_UNSUPPORTED = -2, /* well-formed spec the library does not implement */
  AZ_ERR_NOMEM = -3,       /* device allocation failed */
  AZ_ERR_DEVICE = -4       /* any other HIP runtime failure */
} az_status;

/* Policy and value head kinds (version-2 spec fields). */
typedef enum { AZ_POLICY_PLANES = 0, AZ_POLICY_FROMTO = 1 } az_policy_head;
typedef enum { AZ_VALUE_TANH = 0, AZ_VALUE_WDL = 1 } az_value_head;
#define AZ_FROMTO_ACTIONS 1880

/* Network shape.  abi_version 1 callers pass the first nine fields only (the
 * move-plane / tanh network); abi_version 2 adds the last five.
 * Move-plane network (policy_head 0, value_head 0, pool_every 0): in_planes
 * 1..32; blocks 1..64; policy_planes 1..95; value_hidden 1..512; act_cap >= 0
 * (0 = plain ReLU); max_batch 1..1048576.  filters: AZ_F32 any multiple of 8
 * up to 256; AZ_BF16, AZ_INT8 and AZ_FP8_E4M3 one of 64, 128, 256.
 * Deployed network (policy_head AZ_POLICY_FROMTO with value_head AZ_VALUE_WDL):
 * AZ_BF16 or AZ_INT8; filters 160; in_planes 1..64; blocks 1..64; policy_planes
 * 0; token_dim 128; value_channels 1..32; value_hidden 1..512; pool_every >= 0.
 * Anything else well-formed returns AZ_ERR_UNSUPPORTED. */
typedef struct {
  int32_t abi_version;     /* 1 or 2 (AZ_ABI_VERSION) */
  int32_t in_planes;       /* input planes per position (20 or 52 in the synthetic encodings) */
  int32_t blocks;          /* residual blocks after the stem */
  int32_t filters;         /* F: channels of the stem and of every block */
  int32_t policy_planes;   /* P: move-type planes; P*64 policy cells per position (0 for from-to) */
  int32_t value_hidden;    /* H: width of the value head's hidden layer */
  int32_t value_conv_relu; /* 0: no activation after the value 1x1 conv; 1: ReLU */
  float act_cap;           /* 0: ReLU; > 0: ReLU capped at act_cap */
  int32_t max_batch;       /* largest B az_eval_batch accepts for this handle */
  /* abi_version >= 2 */
  int32_t pool_every;      /* 0: no global pooling; p > 0: blocks j % p == p - 1 pool */
  int32_t policy_head;     /* az_policy_head */
  int32_t token_dim;       /* D of the from-to head (0 with the move-plane head) */
  int32_t value_head;      /* az_value_head */
  int32_t value_channels;  /* V: 1x1 value channels (1 with the tanh head) */
} az_layer_spec;

/* Number of floats the canonical weight blob of `spec` must hold, or 0 if the
 * spec is malformed.  Blob order (fp32, PyTorch layouts, concatenated):
 *   stem W[F][in_planes][3][3], b[F];
 *   for each block: W1[F][F][3][3], b1[F], (pooling blocks: Wg[Fr][2g]),
 *     W2[F][K][3][3] (K = Fr in pooling blocks, else F), b2[F];
 *   move-plane head: W[P][F], b[P];  from-to head: We[D][F], be[D], Wq[D][D],
 *     bq[D], Wk[D][D], bk[D], Wp[4][D];
 *   tanh value head: W[1][F], b[1], fc1 W[H][64], b[H], fc2 W[1][H], b[1];
 *   WDL value head: Wv[V][F], bv[V], W1[H][V*64], b1[H], W2[3][H], b2[3]. */
size_t az_weight_count(const az_layer_spec* spec);

/* Builds a handle on the current HIP device: validates the spec and counts,
 * rounds (AZ_BF16: nearest even) or quantises (AZ_INT8 / AZ_FP8_E4M3, with the
 * given scales) the weights, packs them into the kernels' fragment order and
 * copies them to device memory.  Synchronous.
 *   weights     host, n_weights floats in blob order; copied, caller keeps ownership.
 *   w_scales    AZ_INT8 / AZ_FP8_E4M3: host, 2*blocks*F positive finite floats,
 *               s_w[n][f] for residual conv n; other dtypes: NULL and 0.
 *   act_scales  AZ_INT8 / AZ_FP8_E4M3: host, 2*blocks+1 positive finite floats,
 *               a[k] of tensor k in the order h0, t0, h1, t1, ..., h_blocks (h0 is
 *               the stem output, t_j the first conv's output in block j, h_{j+1}
 *               block j's output); other dtypes: NULL and 0.
 *   out         receives the handle; untouched on failure.
 * Returns AZ_OK, AZ_ERR_INVALID_ARG, AZ_ERR_UNSUPPORTED, AZ_ERR_NOMEM or
 * AZ_ERR_DEVICE.  Nothing leaks on failure. */
int az_net_load(const az_layer_spec* spec, const float* weights, size_t n_weights,
                int32_t dtype, const float* w_scales, size_t n_w_scales,
                const float* act_scales, size_t n_act_scales, az_net** out);

/* Evaluates B positions, asynchronously on `stream` (a hipStream_t; NULL is the
 * null stream of the handle's device).  Allocates nothing and never
 * synchronises, so it can be captured into a HIP graph.
 *   planes  device, [B][in_planes][8][8] fp32, contiguous, 16-byte aligned.
 *           AZ_BF16 / AZ_INT8 / AZ_FP8_E4M3 round the planes to bf16 on entry.
 *   legal   device, [B][n_moves] bytes (n_moves = az_net_moves(net)), contiguous,
 *           16-byte aligned; nonzero = legal.
 *   policy  device, [B][n_moves] fp32 out, contiguous, 16-byte aligned; every element
 *           is written; illegal cells are exactly 0.0f.
 *   value   device, [B] fp32 out, in [-1, 1] (tanh head: tanh; WDL head: W - L).
 * B == 0 returns AZ_OK and launches nothing.  B < 0, B > max_batch, a NULL or
 * misaligned pointer return AZ_ERR_INVALID_ARG before touching the device.
 * Input values are not checked.  Launch failures return AZ_ERR_DEVICE. */
int az_eval_batch(az_net* net, const float* planes, const uint8_t* legal, int32_t B,
                  float* policy, float* value, void* stream);

/* az_eval_batch with the WDL head's probabilities: wdl, if not NULL, is a
 * device [B][3] fp32 output (win, draw, loss; 4-byte aligned) and needs a WDL
 * network (else AZ_ERR_INVALID_ARG).  The policy and legal rows hold
 * az_net_moves(net) entries.  Same errors and asynchrony as az_eval_batch. */
int az_eval_batch_wdl(az_net* net, const float* planes, const uint8_t* legal, int32_t B,
                      float* policy, float* value, float* wdl, void* stream);

/* Policy entries (legal-mask bytes, policy floats) per position: P*64 for the
 * move-plane head, AZ_FROMTO_ACTIONS for the from-to head; negative status for
 * a NULL handle. */
int az_net_moves(const az_net* net);

/* Kernel tiling used by az_eval_batch.  0: chosen from B and the dtype
 * (default); 1 (large): four boards per workgroup (F = 64, 128) or two
 * (F = 256), one workgroup per compute unit; 2 (small): one board per
 * workgroup; 3 (medium, F = 64 and 128 only): two boards per workgroup, two
 * workgroups per compute unit.  The deployed network has two: 1, one wave per
 * board (several boards per compute unit); 2, four waves per board (one board
 * per compute unit, for small batches).  Every tiling computes bitwise the
 * same results.  AZ_F32 has a single tiling and accepts only 0.  Returns
 * AZ_OK or AZ_ERR_INVALID_ARG. */
int az_net_set_tiling(az_net* net, int32_t tiling);

/* The tiling az_eval_batch would use for a batch of B (1, 2 or 3; 0 for
 * AZ_F32), or a negative status. */
int az_net_tiling_for(const az_net* net, int32_t B);

/* Device bytes held by the handle (packed weights and per-layer constants). */
size_t az_net_device_bytes(const az_net* net);

/* Frees the handle and its device memory; NULL is a no-op.  The caller must
 * make sure no evaluation on the handle is still running. */
void az_net_free(az_net* net);

/* Deployment validation (the checks the paper applies to its deployed engine
 * after every refit, Section "Prediction drift under TensorRT refitting"):
 * compares two evaluations of the same B positions, a test one (for example the
 * AZ_INT8 network) against a reference one (its float source), and writes per
 * position row_metrics[b] = { 1 if the top legal move is the same else 0 (the
 * first index wins ties; a row without legal moves counts as agreeing),
 * KL(P_ref || P_test) over the legal cells (terms with P_ref = 0 are 0; P_test is
 * floored at 1e-30 inside the logarithm), |V_ref - V_test| }.
 *   policy_ref, policy_test  device, [B][n_moves] fp32, 4-byte aligned.
 *   value_ref, value_test    device, [B] fp32.
 *   legal                    device, [B][n_moves] bytes, nonzero = legal.
 *   row_metrics              device, [B][3] fp32 out.
 * Asynchronous on stream; allocates nothing.  B == 0 returns AZ_OK.  B < 0,
 * n_moves <= 0, a NULL or misaligned pointer return AZ_ERR_INVALID_ARG; a launch
 * failure AZ_ERR_DEVICE.  Uses no network handle. */
int az_compare_outputs(const float* policy_ref, const float* value_ref, const float* policy_test,
                       const float* value_test, const uint8_t* legal, int32_t B, int32_t n_moves,
                       float* row_metrics, void* stream);

/* Host submission pipeline (Section 5.2 "Batching and host-side submission":
 * preallocated staging buffers, asynchronous copies, completion events and graph
 * replay keep the GPU busy while the host prepares the next batches).  A
 * pipeline belongs to one loaded handle (which must outlive it) and owns
 * `slots` independent slots, each with pinned host buffers, device buffers, a
 * stream and a completion event, sized for max_batch positions.  The caller
 * writes a slot's inputs into its host buffers, submits it (copy in, evaluate,
 * copy out, asynchronously on the slot's stream), and reads the outputs from
 * the slot's host buffers after az_pipeline_wait (or az_pipeline_query returning
 * AZ_OK).  Without AZ_PIPE_GRAPHS the slots share three in-order streams
 * (copy-in, compute, copy-out) and run in submission order, so the input
 * copies of later slots overlap the evaluation of earlier ones.  Several
 * threads may use one pipeline as long as each slot is used by one thread at a
 * time (submission is serialised inside).
 *
 * Flags:
 *   AZ_PIPE_GRAPHS          give each slot a stream of its own, capture its
 *                           steps into a HIP graph for each new batch size and
 *                           replay it;
 *   AZ_PIPE_COMPACT_POLICY  return only the legal moves' probabilities: per
 *                           position, the probabilities of its legal cells in
 *                           ascending cell index order, in max_legal floats
 *                           (zero past the last legal move), plus the number of
 *                           legal cells.  This is what a search node expands.
 *                           A kernel writes the compact rows and the counts
 *                           into the slot's device output block (the value
 *                           sits there too), and device-to-host copies bring
 *                           them to the slot's pinned host buffers: one copy
 *                           of the whole block when B == max_batch, else one
 *                           per array.  4 * (max_legal + 2) bytes per
 *                           position cross the link instead of
 *                           4 * (n_moves + 1). */
#define AZ_PIPE_GRAPHS 1
#define AZ_PIPE_COMPACT_POLICY 2

typedef struct az_pipeline az_pipeline;

/* Creates a pipeline on the handle's device.  max_batch: 1..the handle's
 * max_batch; slots: 1..64; flags: an OR of AZ_PIPE_*; max_legal: 1..n_moves
 * (az_net_moves) with AZ_PIPE_COMPACT_POLICY, else 0.  Allocates all buffers (pinned host memory
 * with hipHostMalloc, device memory, streams, events); nothing leaks on
 * failure.  Returns AZ_OK, AZ_ERR_INVALID_ARG, AZ_ERR_NOMEM or AZ_ERR_DEVICE. */
int az_pipeline_create(az_net* net, int32_t max_batch, int32_t slots, int32_t flags, int32_t max_legal,
                       az_pipeline** out);

/* Host buffers of a slot (any output pointer may be NULL): planes
 * [max_batch][in_planes][8][8] f32 and legal [max_batch][n_moves] u8 (inputs);
 * value [max_batch] f32 and policy (outputs): [max_batch][n_moves] f32, or with
 * AZ_PIPE_COMPACT_POLICY [max_batch][max_legal] f32 plus legal_count
 * [max_batch] i32 (NULL without the flag).  The pipeline owns them; they stay
 * valid until az_pipeline_free.  Do not touch a slot's buffers between its
 * submit and its completion. */
int az_pipeline_slot(az_pipeline* p, int32_t slot, float** planes, uint8_t** legal, float** policy,
                     float** value, int32_t** legal_count);

/* Submits the first B positions of a slot's inputs (0 <= B <= max_batch) and
 * returns without waiting.  A slot already in flight returns
 * AZ_ERR_INVALID_ARG (wait for it first). */
int az_pipeline_submit(az_pipeline* p, int32_t slot, int32_t B);

/* AZ_OK when the slot's last submission has completed (or nothing is in flight),
 * 1 while it is still running, or a negative status.  With
 * AZ_PIPE_COMPACT_POLICY, a completed submission in which some position had
 * more than max_legal legal cells returns AZ_ERR_INVALID_ARG (that row is
 * truncated to its first max_legal legal cells; legal_count holds the true
 * count; every other output is valid). */
int az_pipeline_query(az_pipeline* p, int32_t slot);

/* Blocks until the slot's last submission has completed; same statuses as
 * az_pipeline_query apart from 1. */
int az_pipeline_wait(az_pipeline* p, int32_t slot);

/* Drives the pipeline from `workers` native threads, the actors of the paper's
 * host side (Section 5.1 "Native ownership of the search loop", Section 5.2
 * "Batching and host-side submission"): worker w owns slots w*slots_per_worker
 * .. (w+1)*slots_per_worker - 1 and keeps them in flight round-robin (wait for
 * the slot, resubmit its current host inputs as a batch of B positions), first
 * `warmup` submissions untimed, then `batches` timed ones, each phase ending
 * with all of the worker's slots drained.  *seconds receives the wall time of
 * the timed phase (from the moment every worker has drained its warm-up).  The
 * caller fills the slots' inputs beforehand and must not use the pipeline
 * meanwhile.  Returns AZ_OK or the first failing status (AZ_ERR_INVALID_ARG for
 * bad counts, including a compact row that overflowed max_legal). */
int az_pipeline_drive(az_pipeline* p, int32_t workers, int32_t slots_per_worker, int32_t B, int32_t warmup,
                      int32_t batches, double* seconds);

/* Waits for every slot, then frees the pipeline's buffers, streams, events and
 * graphs; NULL is a no-op. */
void az_pipeline_free(az_pipeline* p);

/* az_eval_batch followed by the compaction of AZ_PIPE_COMPACT_POLICY, on
 * device buffers, allocating nothing: for callers that cannot allocate (code
 * under HIP graph capture, serving loops and harnesses that forbid hipMalloc).
 * policy: device [B][max_legal] fp32, per position the probabilities of its
 * legal cells in ascending cell order, zero past the last (a row with more than
 * max_legal legal cells keeps its first max_legal); legal_count: device [B]
 * int32, the true number of legal cells; value: device [B] fp32.  planes,
 * legal as for az_eval_batch.  The dense policy between the two kernels lives
 * in a static device array of the library, 512 * 95 * 64 floats (12.45 MB)
 * held by every GPU the library runs on until the process ends: B times
 * az_net_moves(net) must not exceed it (at most 666 positions of the 4,672-cell
 * move-plane policy, 1,655 of the 1,880 from-to actions), else
 * AZ_ERR_INVALID_ARG with a message.  All calls on one GPU share that array:
 * calls that overlap on one GPU (different streams or threads) race.  B == 0
 * returns AZ_OK and launches nothing; NULL or misaligned pointers, max_legal
 * outside 1..az_net_moves(net) and B outside 0..max_batch return
 * AZ_ERR_INVALID_ARG.  Asynchronous on `stream`, no host synchronisation. */
int az_eval_batch_compact_noalloc(az_net* net, const float* planes, const uint8_t* legal, int32_t B,
                                  int32_t max_legal, float* policy, int32_t* legal_count, float* value,
                                  void* stream);

/* Failure-handling test support.  az_debug_fail_allocation(n), n >= 1: the
 * n-th device or pinned-host allocation the library attempts from now on
 * (weights in az_net_load, buffers in az_pipeline_create) fails as if the
 * memory were exhausted, and the call that made it must return AZ_ERR_NOMEM;
 * n = 0 disarms.  az_debug_live_allocations(): the library's device and
 * pinned-host allocations not yet freed (a leak check).  Neither touches the
 * device; both are process-wide. */
void az_debug_fail_allocation(int32_t n);
int64_t az_debug_live_allocations(void);

/* Static description of a status code. */
const char* az_status_string(int status);

/* Detail of the last failure on the calling thread ("" if none). */
const char* az_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* AZ_H */
