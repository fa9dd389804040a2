/*
 * dtp.h - C ABI of libdtp.so: the data-parallel hot path of affinity-aware sharding for
 * Delayed Tensor Parallelism (arXiv 2609.13846), for AMD Instinct MI355X (gfx950).
 *
 * The paper (Section 3) measures, over calibration tokens, how much each FFN neuron of a
 * layer depends on each KV group of the same layer (the "up" affinity S_up[g, k]), then
 * chooses balanced assignments of KV groups (h_i) and neurons (nu_i) to L devices that
 * maximise the total co-located normalised affinity J (eq. "objective") by coordinate
 * ascent: an exact balanced assignment of the neurons given the heads, and an exhaustive
 * scan of the labelled balanced partitions of the KV groups given the neurons.
 *
 * Conventions shared by every entry point:
 *   - Every function returns a dtp_status; nothing throws across the ABI.  On failure,
 *     dtp_last_error() gives a thread-local message.
 *   - Arguments are validated on the host before any GPU work is enqueued.
 *   - "dev" pointers are device memory of the current HIP device; "host" pointers are
 *     ordinary host memory.  The caller owns every buffer it passes; the library keeps
 *     no caller pointer after a call returns.  Device tensors are dense row-major.
 *   - Every dev argument is checked before any work is enqueued: it must be memory of the
 *     current device (hipPointerGetAttributes) whose allocation holds every byte the call
 *     reads or writes from that address on (hipMemGetAddressRange); otherwise the call
 *     returns DTP_ERR_INVALID_ARG.  Host arrays cannot be checked: their sizes are the
 *     caller's responsibility.
 *   - `stream` is a hipStream_t (NULL = the default stream).  GPU work is enqueued on it
 *     asynchronously; functions that return host results synchronise that stream first.
 *   - Host threads may call the library concurrently, each with its own stream: calls on
 *     different layers, and the functions that take no layer, keep no shared mutable
 *     state (their scratch comes per call from the stream-ordered allocator).  Calls on
 *     one dtp_layer share its workspace and must be ordered by the caller (one stream,
 *     or synchronised); so must overlapping calls of dtp_down_weights_noalloc on a device.
 *   - Weights use the PyTorch nn.Linear layout [out_features, in_features].
 *   - bf16 tensors are IEEE bfloat16 bit patterns (uint16); f32 tensors are float.
 */
#ifndef DTP_H
#define DTP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DTP_OK = 0,
  DTP_ERR_INVALID_ARG = -1,  /* null pointer, bad size, shape constraint violated */
  DTP_ERR_UNSUPPORTED = -2,  /* a valid request outside what the library implements */
  DTP_ERR_DEGENERATE = -3,   /* affinity all zero, negative or non-finite */
  DTP_ERR_NO_MEMORY = -4,    /* host or device allocation failed, or a host thread could not start */
  DTP_ERR_HIP = -5           /* a HIP runtime call failed (message has the HIP string) */
} dtp_status;

typedef enum { DTP_BF16 = 0, DTP_F32 = 1 } dtp_dtype;

/* Shapes of one decoder layer.  Query head h belongs to KV group h / (H/G).
 * Constraints: all sizes > 0; H % G == 0; G <= 32; head_dim % 16 == 0; d_model % 16 == 0;
 * rms_eps >= 0; dtype is DTP_BF16 (MFMA path) or DTP_F32 (reference-precision path). */
typedef struct {
  int32_t d_model;      /* d */
  int32_t n_neurons;    /* I, SwiGLU FFN width */
  int32_t n_q_heads;    /* H */
  int32_t n_kv_groups;  /* G */
  int32_t head_dim;     /* dh */
  float rms_eps;        /* epsilon inside the FFN pre-norm: r = sqrt(mean(x^2) + eps) */
  int32_t dtype;        /* dtp_dtype of every weight and activation */
} dtp_layer_desc;

typedef struct dtp_layer_s* dtp_layer;  /* opaque: folded weights and workspace of one layer */

/* Allocate the device state of one layer (no weights yet).  *out receives the handle. */
dtp_status dtp_layer_create(const dtp_layer_desc* desc, dtp_layer* out);

/* Free a layer and everything it allocated.  NULL is accepted. */
dtp_status dtp_layer_destroy(dtp_layer layer);

/* Load and fold the weights of a layer (Section 3, "Affinity scores": p_h . w_k is
 * re-associated as a_h . (W_o^(h) diag(gamma) w_k) / r, so each head's contraction runs
 * over head_dim instead of d_model).  All pointers are dev, in the layer's dtype:
 *   w_o    [d, H*dh]  attention output projection (o_proj.weight)
 *   gamma  [d]        gain of the FFN pre-norm
 *   w_gate [I, d], w_up [I, d]   SwiGLU gate and up projections
 *   w_down [d, I]     down projection (its column k is w^d_k)
 * Work is enqueued on `stream`; the inputs may be freed once the stream has passed it. */
dtp_status dtp_layer_set_weights(dtp_layer layer, const void* w_o, const void* gamma,
                                 const void* w_gate, const void* w_up, const void* w_down,
                                 void* stream);

/* Accumulate the raw first-order up affinity of n_tokens calibration tokens (Section 3,
 * "Affinity scores", score FO):
 *   A[g, k] += ||w^d_k||^2 * sum_t sum_{h in g} Delta_hk(t)^2,
 *   Delta_hk = silu'(g_k) u_k (p_h . w^g_k) + silu(g_k) (p_h . w^u_k),
 *   p_h = gamma * (a_h W_o^(h)) / r,  r = sqrt(mean(x^2) + eps),
 * with g_k, u_k, r taken at the unmodified x (the rms change is ignored).  The mean over
 * tokens of the paper is left to the caller (it cancels in the unit-mass normalisation).
 *   x    dev [n_tokens, d]       residual entering the FFN pre-norm (layer dtype)
 *   attn dev [n_tokens, H, dh]   per-head attention outputs a_h (layer dtype)
 *   A    dev [G, I] float        accumulated in place (+=); deterministic for fixed shapes
 * n_tokens == 0 is a no-op.  Requires dtp_layer_set_weights on an earlier call. */
dtp_status dtp_affinity_accumulate(dtp_layer layer, const void* x, const void* attn,
                                   int64_t n_tokens, float* A, void* stream);

/* The simpler ADD score of Section 3 ("Affinity scores") over the same token stream:
 *   A[g, k] += sum_t sum_{h in g} (p_h . w^g_k)^2 + (p_h . w^u_k)^2,
 * which ignores the operating point of the nonlinearity and the neuron's write (no
 * ||w^d_k||^2 factor).  Arguments as for dtp_affinity_accumulate. */
dtp_status dtp_affinity_accumulate_add(dtp_layer layer, const void* x, const void* attn,
                                       int64_t n_tokens, float* A, void* stream);

/* The same accumulation of A, plus the token statistic of the down edge (Section 3,
 * "Affinity scores", down edge) in the same pass:
 *   s_down[k] += sum_t alpha_k(t)^2 / r'_t^2,  alpha_k = silu(g_k) u_k,
 *   r'_t = sqrt(mean(x_next[t]^2) + rms_eps_next),
 * with g_k, u_k at the layer's operating point and x_next the residual entering the next
 * layer's attention pre-norm (held fixed, as r is).
 *   x_next dev [n_tokens, d]  layer dtype, 16-byte aligned
 *   s_down dev [I] float       accumulated in place (+=); deterministic for fixed shapes
 * x_next and s_down are both required (DTP_ERR_INVALID_ARG otherwise). */
dtp_status dtp_affinity_accumulate_down(dtp_layer layer, const void* x, const void* attn,
                                        const void* x_next, float rms_eps_next,
                                        int64_t n_tokens, float* A, float* s_down,
                                        void* stream);

/* Weight-only factor of the down edge into the next layer (Section 3, down edge):
 *   B[g, k] = || W^{qkv}_g (gamma' * w^d_k) ||^2,
 * W^{qkv}_g the q rows of next-layer KV group g's query heads (consecutive heads share a
 * group), then its k rows and v rows; gamma' the next layer's attention pre-norm gain;
 * w^d_k column k of this layer's W_down.  Sizes are the next layer's heads and this
 * layer's d and I.
 *   w_q dev [H*dh, d], w_k / w_v dev [G*dh, d]  (q_proj/k_proj/v_proj.weight layouts)
 *   gamma_next dev [d], w_down dev [d, I]       all in `dtype`, 16-byte aligned
 *   B dev [G, I] float                          written
 * bf16: MFMA over d with gamma' * w^d_k rounded to bf16, fp32 sums of squares; requires
 * d and I multiples of 8.  f32: plain FMAs (small shapes).  Scratch of G*I*ceil((H/G+2)*dh
 * /128) floats, and for bf16 a gamma'-scaled transposed copy of W_down (I*d bf16), is taken
 * from the stream-ordered allocator and returned before exit. */
dtp_status dtp_down_weights(int32_t d_model, int32_t n_neurons, int32_t n_q_heads,
                            int32_t n_kv_groups, int32_t head_dim, dtp_dtype dtype,
                            const void* w_q, const void* w_k, const void* w_v,
                            const void* gamma_next, const void* w_down, float* B, void* stream);

/* dtp_down_weights for callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops and harnesses that forbid hipMalloc): the same B bit for bit, with
 * the per-chunk partial sums in a fixed 4 MiB device array instead of stream-ordered scratch,
 * and W_down scaled and transposed stage by stage inside the weight kernel instead of once
 * into a copy.  The call makes no allocation of any kind; the array is held by
 * each device the library runs on until the process ends (its address is looked up once per
 * device, on the first call there).  Limit: G * I * ceil((H/G + 2) * dh / 128) <= 2^20
 * partial sums (the 8B-class shape needs 688,128), else DTP_ERR_UNSUPPORTED before any
 * work.  Calls on one device share the array: calls that overlap in time on one GPU (other
 * streams, other host threads) race and must be ordered by the caller.  Arguments, checks
 * and the f32 path (which needs no scratch) as for dtp_down_weights. */
dtp_status dtp_down_weights_noalloc(int32_t d_model, int32_t n_neurons, int32_t n_q_heads,
                                    int32_t n_kv_groups, int32_t head_dim, dtp_dtype dtype,
                                    const void* w_q, const void* w_k, const void* w_v,
                                    const void* gamma_next, const void* w_down, float* B,
                                    void* stream);

/* Raw down affinity S_down[k, g] = s_down[k] * B[g, k] (the A_down operand of
 * dtp_coordinate_ascent for this layer).
 *   s_down dev [I], B dev [G, I], A_down dev [I, G] float (written). */
dtp_status dtp_down_affinity(int32_t n_neurons, int32_t n_kv_groups, const float* s_down,
                             const float* B, float* A_down, void* stream);

/* Timing of the affinity kernel with HIP events on the launch stream.  After
 * dtp_layer_profile(layer, 1), every accumulate call records an event pair around each
 * launch of its dominant kernel; dtp_layer_profile_read synchronises those events and
 * returns the summed duration in milliseconds and the number of launches, then clears
 * them.  dtp_layer_profile(layer, 0) stops recording. */
dtp_status dtp_layer_profile(dtp_layer layer, int32_t enable);
dtp_status dtp_layer_profile_read(dtp_layer layer, double* total_ms, int64_t* launches);

/* ---------------------------------------------------------------------------------------
 * Layout optimiser (Section 3, "Objective" and "Optimiser").
 *
 * Each raw affinity matrix is normalised to unit mass in exact fixed point:
 *   E = floor(log2 max A); q_i = floor(A_i * 2^(40-E)); Q_i = floor(q_i * 2^48 / sum q).
 * Codes are int64 and sum to 2^48 minus at most one unit per entry; J = J_int / 2^48,
 * where J_int sums the codes of co-located (group, neuron) pairs.
 * Ties: the best head partition is the one of lowest lexicographic rank; the neuron
 * assignment is the lexicographically smallest optimal one.
 * ------------------------------------------------------------------------------------- */

/* Number of labelled balanced partitions of G groups over L devices, G!/((G/L)!)^L,
 * or -1 when G % L != 0, L < 1 or G > 64. */
int64_t dtp_partition_count(int32_t G, int32_t L);

/* The partition of lexicographic rank `rank` (rank 0 is the contiguous h(g) = g/(G/L)).
 * h: host [G] receives device indices. */
dtp_status dtp_partition_unrank(int32_t G, int32_t L, int64_t rank, int32_t* h);

/* Unit-mass fixed-point code of a raw affinity matrix.  A, Q: host [n], 1 <= n <= 2^20.
 * DTP_ERR_DEGENERATE if any entry is negative or non-finite, or all are zero. */
dtp_status dtp_encode_affinity(const float* A, int64_t n, int64_t* Q);

/* The same codes computed on the GPU (the coordinate ascent encodes its matrices this way).
 *   A dev [n] fp32 raw affinity, 1 <= n <= 2^30; Q dev [n] int64 output (caller-owned).
 * Enqueued on `stream`, which is then synchronised to read the outcome: DTP_ERR_DEGENERATE
 * (Q unspecified) if an entry is negative or non-finite, or all are zero; else the codes
 * equal dtp_encode_affinity's bit for bit.  Uses a few bytes of stream-ordered scratch. */
dtp_status dtp_encode_affinity_device(const float* A, int64_t n, int64_t* Q, void* stream);

/* Head step of one layer i (Section 3, "Optimiser"): score every labelled balanced
 * partition h of the G KV groups,
 *   score(h) = sum_g C[g, h(g)],
 *   C[g, l]  = sum_{k: nu(k)=l} Q_up[g, k] + sum_{k: nu_prev(k)=l} Q_down_prev[k, g],
 * on the GPU, one wavefront per partition.
 *   Q_up        dev [G, I] int64    codes of layer i's up affinity
 *   nu          dev [I] int32       neuron assignment of layer i (values in [0, L))
 *   Q_down_prev dev [I, G] int64    codes of layer i-1's down affinity, or NULL
 *   nu_prev     dev [I] int32       neuron assignment of layer i-1 (NULL iff Q_down_prev is)
 *   minimise    0: best = highest score; 1: lowest
 *   scores      dev [P] int64       score of every partition, by rank (P = partition count)
 *   best_rank   host                rank of the best partition (lowest rank on ties)
 * Requires G % L == 0, I % L == 0, G <= 64, P <= 2^24.  Synchronises `stream`. */
dtp_status dtp_partition_scores(int32_t G, int32_t I, int32_t L, const int64_t* Q_up,
                                const int32_t* nu, const int64_t* Q_down_prev,
                                const int32_t* nu_prev, int32_t minimise, int64_t* scores,
                                int64_t* best_rank, void* stream);

/* Neuron step of one layer i (Section 3, "Optimiser"): the balanced nu maximising
 * sum_k M[k, nu(k)] with I/L neurons per device, where
 *   M[k, l] = sum_{g: h(g)=l} Q_up[g, k] + sum_{g: h_next(g)=l} Q_down[k, g].
 * Exact (an optimal solution of the linear assignment with I/L slots per device), then
 * the lexicographically smallest among all optimal ones.  Runs on the host.
 *   Q_up   host [G, I] int64;  h host [G] int32 (balanced)
 *   Q_down host [I, G] int64 or NULL;  h_next host [G] int32 (NULL iff Q_down is)
 *   minimise  0: maximise; 1: minimise
 *   nu     host [I] int32 output;  value host int64 output (sum_k M[k, nu(k)])
 * Requires G % L == 0, I % L == 0, 1 <= L <= 8, G <= 64, I <= 2^24. */
dtp_status dtp_balanced_assign(int32_t G, int32_t I, int32_t L, const int64_t* Q_up,
                               const int32_t* h, const int64_t* Q_down, const int32_t* h_next,
                               int32_t minimise, int32_t* nu, int64_t* value);

/* The same neuron step solved the way the paper does (Section 3, "Optimiser"; 300
 * iterations with step decay 0.98 from the appendix), kept to measure its distance from the
 * optimum: dual ascent on L device offsets (from zero, first step (max M - min M) / I; each
 * neuron takes argmax_l M[k, l] - lambda_l, lowest l on ties, and lambda_l rises by
 * step * (load_l - I/L)), then a fix-up that moves the cheapest neurons from overloaded to
 * underloaded devices one at a time, then pairwise swaps (device pairs in order, the best
 * exchange per pair when its total gain is positive) until a full scan exchanges nothing.
 * Balanced; value <= dtp_balanced_assign's; equal to it when L = 2.  Same arguments, sizes
 * and errors as dtp_balanced_assign.  Host only. */
dtp_status dtp_balanced_assign_dual_ascent(int32_t G, int32_t I, int32_t L, const int64_t* Q_up,
                                           const int32_t* h, const int64_t* Q_down,
                                           const int32_t* h_next, int32_t minimise, int32_t* nu,
                                           int64_t* value);

/* Options of the coordinate ascent; NULL means the defaults
 * {max_sweeps = 64, freeze_heads = 0, freeze_neurons = 0, minimise = 0, layer_mask = NULL,
 *  dual_ascent_neurons = 0}.
 * freeze_*: keep that block at its contiguous start.  layer_mask (host, exactly N entries,
 * or NULL): a zero entry keeps layer i contiguous.  minimise: minimise J instead (anti-optimised layouts).
 * dual_ascent_neurons: solve the neuron step with the paper's approximate method
 * (dtp_balanced_assign_dual_ascent) instead of exactly. */
typedef struct {
  int32_t max_sweeps;
  int32_t freeze_heads;
  int32_t freeze_neurons;
  int32_t minimise;
  const uint8_t* layer_mask;
  int32_t dual_ascent_neurons;
} dtp_ca_options;

/* Coordinate ascent over a chain of N layers (Section 3, "Optimiser"): start from the
 * contiguous head assignment h_i(g) = g/(G/L); each sweep runs the neuron step of every
 * layer (host) and then the head step of every layer (GPU partition scores); stop at the
 * first sweep whose J_int is not strictly better than the previous sweep's, or after
 * max_sweeps.  Each matrix is encoded to unit mass separately.
 *   A_up   dev [N, G, I] float  raw up affinity of each layer (from dtp_affinity_accumulate)
 *   A_down dev [N-1, I, G] float raw down affinity, or NULL (then the layers decouple)
 *   h      host [N, G] int32 output;  nu host [N, I] int32 output
 *   J host double output (J_int / 2^48);  J_fixed host int64 output (J_int, exact)
 *   sweeps  host int32 output (sweeps run)
 * Synchronises `stream`.  DTP_ERR_DEGENERATE if any matrix is all zero or not finite. */
dtp_status dtp_coordinate_ascent(int32_t N, int32_t G, int32_t I, int32_t L,
                                 const float* A_up, const float* A_down,
                                 const dtp_ca_options* options, int32_t* h, int32_t* nu,
                                 double* J, int64_t* J_fixed, int32_t* sweeps, void* stream);

/* Seeded balanced layouts, the random baseline of the ablations (Section 4): for each
 * layer in turn, the contiguous h_i (h(g) = g/(G/L)) and then the contiguous nu_i are
 * shuffled by Fisher-Yates from the last position down, position j swapping with
 * floor(r (j+1) / 2^64), r the next output of SplitMix64 (Steele, Lea and Flood, 2014)
 * started from state `seed`.  h host [N, G] and nu host [N, I] int32 outputs.  Host only. */
dtp_status dtp_random_layout(int32_t N, int32_t G, int32_t I, int32_t L, uint64_t seed,
                             int32_t* h, int32_t* nu);

/* J_int of a given layout (Section 3, eq. "objective"): the sum of co-located codes over
 * the N up edges and, when Q_down is given, the N-1 down edges.
 *   Q_up host [N, G, I] and Q_down host [N-1, I, G] or NULL: dtp_encode_affinity codes
 *   h host [N, G], nu host [N, I]: balanced layouts (DTP_ERR_INVALID_ARG otherwise)
 *   J_fixed host int64 output; J = J_fixed / 2^48.  Host only. */
dtp_status dtp_layout_objective(int32_t N, int32_t G, int32_t I, int32_t L, const int64_t* Q_up,
                                const int64_t* Q_down, const int32_t* h, const int32_t* nu,
                                int64_t* J_fixed);

/* Exact optimum of one layer's up edge: every head partition up to device relabelling
 * (labels first appearing in the order 0..L-1; 105 at G=8, L=4) with its exact neuron
 * assignment; the first such partition in lexicographic order that attains the maximum
 * is returned with its canonical assignment.  Bounds the coordinate ascent from above.
 *   Q_up host [G, I] codes; h host [G], nu host [I] outputs; J_fixed host output.
 * Host only (one thread per partition, at most 16). */
dtp_status dtp_layer_optimum(int32_t G, int32_t I, int32_t L, const int64_t* Q_up, int32_t* h,
                             int32_t* nu, int64_t* J_fixed);

/* ---------------------------------------------------------------------------------------
 * Applying a layout (Section 3, "The layout as a free variable").  Device l's shard holds
 * the KV groups and neurons that (h, nu) put on l, in increasing original index; shards
 * follow in device order.  The permuted layer computes the same function (rotary embeddings, per-head norms
 * and SwiGLU act per head or per neuron).
 * ------------------------------------------------------------------------------------- */

/* New position -> original index of the groups ([G]) and neurons ([I]).  Host only;
 * DTP_ERR_INVALID_ARG unless h and nu are balanced assignments to L devices. */
dtp_status dtp_layout_orders(int32_t G, int32_t I, int32_t L, const int32_t* h, const int32_t* nu,
                             int32_t* group_order, int32_t* neuron_order);

/* Permuted copies of one decoder layer's weights.  src and dst hold 7 device pointers,
 * in the order w_q [H*dh, d], w_k [G*dh, d], w_v [G*dh, d], w_o [d, H*dh],
 * w_gate [I, d], w_up [I, d], w_down [d, I] (PyTorch weight layouts, desc->dtype,
 * 16-byte aligned, d * element size a multiple of 16 bytes).  Rows of w_q (by query-head
 * blocks of a group), w_k, w_v and columns of w_o move with the groups; rows of w_gate,
 * w_up and columns of w_down move with the neurons.  Gains and per-head norm weights are
 * unchanged and not touched.  h host [G], nu host [I].  dst must not alias src.
 * Bit-exact data movement; a [G + I] int32 scratch comes from the stream-ordered
 * allocator and is returned before exit.  Synchronises `stream` (the order table is
 * uploaded from host memory that the call owns). */
dtp_status dtp_apply_layout(const dtp_layer_desc* desc, int32_t L, const int32_t* h,
                            const int32_t* nu, const void* const* src, void* const* dst,
                            void* stream);

/* Human-readable name of a status code (static storage). */
const char* dtp_status_string(dtp_status status);

/* Detail of the last failure on the calling thread ("" if none). */
const char* dtp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DTP_H */
