/*
 * d2moe.h -- C ABI of the MI355X (gfx950) MoE-layer hot path of D^2MoE
 * (dual routing + matryoshka weight quantization, arXiv 2504.15299).
 *
 * One MoE layer forward under dual routing: every token gets its top-k expert
 * IDs, every activated expert gets a bit-width from a per-(request, expert)
 * table (Fig. 1: expert ID *and* bit-width), and each expert's SwiGLU FFN
 * reads its nested MWQ weights (Sec. 3.3) only up to that bit-width.
 *
 * Conventions for every entry point
 *  - Pointers named as device buffers are caller-owned device memory (HIP);
 *    the library never allocates, frees or keeps them, so calls on different
 *    streams are independent.  The one piece of global state is the fixed
 *    scratch array of d2moe_moe_forward_noalloc (one per GPU, process
 *    lifetime).
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    All argument checks run on the host before any launch; on failure a
 *    negative status is returned and nothing is launched.  Work after a
 *    successful return is asynchronous on `stream`; a launch failure is
 *    reported as D2MOE_EHIP.  Nothing here synchronizes with the host.
 *  - Shapes: a weight matrix is [rows][cols] with groups of `group`
 *    consecutive columns (the reduction dimension); group is 64 or 128,
 *    cols % group == 0 and rows % (2048/group) == 0.  Bit-width ladder
 *    1 <= b_min <= b_max <= 8, one bit per step (Sec. 3.3.1).
 */
#ifndef D2MOE_H
#define D2MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t d2moe_status;
enum {
  D2MOE_OK = 0,
  D2MOE_EINVAL = -1,        /* bad argument (shape, null pointer, range) */
  D2MOE_EUNSUPPORTED = -2,  /* valid but not implemented (e.g. dtype) */
  D2MOE_EHIP = -3,          /* a HIP launch or runtime call failed */
  D2MOE_EWORKSPACE = -4,    /* workspace missing or smaller than required */
  D2MOE_ESCRATCH = -5       /* sizes need more than the fixed no-allocation
                               scratch of d2moe_moe_forward_noalloc */
};

/* Bytes of the fixed per-GPU scratch array of d2moe_moe_forward_noalloc. */
#define D2MOE_NOALLOC_SCRATCH_BYTES (32u << 20)

typedef enum { D2MOE_F32 = 0, D2MOE_BF16 = 1 } d2moe_dtype;

/* Human-readable name of a status code (static string, never NULL). */
const char* d2moe_status_string(d2moe_status s);

/*
 * Packed MWQ weights of n_experts matrices of [rows][cols] (Sec. 3.3.1,
 * DS: nested codes Q_b1, residual sign planes, per-group scales and zeros).
 * Canonical tiled bit-plane layout, experts outermost, BR = 2048/group rows
 * per block, KB = cols/group blocks per block-row, levels = b_max-b_min+1:
 *   planes [E][rows/BR][KB][b_max][64] uint32: plane p < b_min holds bit p of
 *          the base code, plane p >= b_min holds the residual sign of
 *          bit-width p+1 (1 = +1); word w of a (block, plane) covers row
 *          w % BR of the block and columns 32*(w/BR) .. +31 of the group,
 *          bit j <-> column 32*(w/BR)+j.  A b-bit read touches planes 0..b-1
 *          only, so lower bit-widths are prefixes of higher ones.
 *   scales [E][rows/BR][KB][levels][BR] binary16: level 0 = base scale s_b1,
 *          level l = residual scale of bit-width b_min+l;
 *   zeros  [E][rows/BR][KB][BR] uint8: integer zero point of the base code.
 * All three are device buffers of the sizes reported by d2moe_mwq_size.
 */
typedef struct {
  int32_t n_experts, rows, cols, group, b_min, b_max;
  uint32_t* planes;
  uint16_t* scales;
  uint8_t* zeros;
} d2moe_mwq;

/*
 * Byte sizes of the three packed buffers (Sec. 3.3.1: one nested tensor per
 * matrix holds the base codes, one sign plane per further bit and the
 * per-group scales and zero points of Eq. 2 and Eq. 4-5, so every bit-width
 * of the ladder is stored once).  Pure host function; returns D2MOE_EINVAL
 * for shapes or ladders the layout does not allow.
 */
d2moe_status d2moe_mwq_size(int32_t n_experts, int32_t rows, int32_t cols,
                            int32_t group, int32_t b_min, int32_t b_max,
                            size_t* planes_bytes, size_t* scales_bytes,
                            size_t* zeros_bytes);

/*
 * MWQ quantize + pack (Sec. 3.3.1: Eq. 2 asymmetric base level, Eq. 4-5
 * binary residual levels, Algorithm 1 with X = I, i.e. no calibration
 * activations).  W: device [n_experts][rows][cols] binary32 (w_dtype must be
 * D2MOE_F32).  Per (row, group): base scale = binary16 of
 * (max(0,max W) - min(0,min W)) / (2^b_min - 1), zero = rint(-min/scale)
 * clamped, codes = clamp(rint(W/scale + zero)); for every further bit:
 * scale = binary16 of mean |residual|, sign plane = [residual >= 0], residual
 * -= scale * sign.  Binary32 arithmetic without contraction, identical to the
 * CPU reference bit for bit.  `out` describes caller-allocated buffers.
 */
d2moe_status d2moe_pack_mwq(const void* W, d2moe_dtype w_dtype,
                            const d2moe_mwq* out, void* stream);

/*
 * Calibration-aware MWQ, step 1 (Algorithm 1, first line): the factor H^c
 * of the regularised Hessian of the calibration activations,
 *     H = 2 X X^T + lambda I,   U upper triangular with H^-1 = U^T U,
 * computed in binary64 (Cholesky factorization of the order-reversed H and
 * a triangular inverse) and stored rounded to binary32.
 *   X:  device [tokens][h] float, calibration activations of the matrix's
 *       input (one row per token; X of the paper is its transpose);
 *   U:  device [h][h] float, written in full (zeros below the diagonal);
 *   info: device int32, 0 on success, else the 1-based column at which H
 *       was found not positive definite (the output is then meaningless);
 *   workspace: device, at least d2moe_mwq_calib_factor_workspace bytes,
 *       256-byte aligned.
 * h % 64 == 0, tokens >= 0, lambda >= 0 (lambda > 0 keeps H definite).
 */
d2moe_status d2moe_mwq_calib_factor_workspace(int32_t h, size_t* bytes);
d2moe_status d2moe_mwq_calib_factor(const float* X, int32_t tokens, int32_t h, double lambda,
                                    float* U, int32_t* info, void* workspace, size_t ws_bytes,
                                    void* stream);

/*
 * Calibration-aware MWQ, step 2 (Sec. 3.3.1, Eq. 3 and Eq. 5 with
 * calibration activations; Algorithm 1's block-level compensation): quantize
 * and pack like d2moe_pack_mwq, but column block by column block (`gamma`
 * columns, 64 or 128, a multiple of the group), moving each block's error
 * onto the later columns of its row before they are quantized:
 *     E = D U_BB^-1,   T_F <- T_F - E U_BF,
 * with D the block's quantization error, U the factor of step 1 (device
 * [cols][cols] float, upper triangle read) shared by all experts of `out`.
 * Every bit-width level is one such pass, restarting from the residual of
 * the levels below, which stay fixed, so lower bit-widths remain prefixes.
 * The codes follow one defined binary32 operation sequence (fmaf chains in
 * ascending index order) and equal the CPU definition bit for bit; with a
 * diagonal U they equal d2moe_pack_mwq's.  W: device [E][rows][cols] float;
 * workspace: at least d2moe_pack_mwq_calibrated_workspace bytes, 256-byte
 * aligned.
 */
d2moe_status d2moe_pack_mwq_calibrated_workspace(int32_t rows, int32_t cols, int32_t gamma,
                                                 size_t* bytes);
d2moe_status d2moe_pack_mwq_calibrated(const void* W, d2moe_dtype w_dtype, const float* U,
                                       int32_t gamma, const d2moe_mwq* out, void* workspace,
                                       size_t ws_bytes, void* stream);

/*
 * Test hook: unpack expert `expert` of `w` at bit-width `bits` into the
 * integer codes of Eq. 2 (base code Q_b1) and Eq. 4 (residual signs of the
 * bit-widths b_min+1 .. bits), with the device decoding routine the forward
 * kernels use.
 *   q1    device [rows][cols] uint8, base codes;
 *   signs device [bits-b_min][rows][cols] int8 (+1/-1), may be NULL when
 *         bits == b_min.
 */
d2moe_status d2moe_debug_unpack(const d2moe_mwq* w, int32_t expert,
                                int32_t bits, uint8_t* q1, int8_t* signs,
                                void* stream);

/*
 * Outputs of the dual router (Fig. 1), all caller-owned device buffers:
 *   logits        [T][E] float   gate logits (x W_g^T + bias, fp32 accumulate)
 *   topk_idx      [T][k] int32   experts, largest logit first, ties to the
 *                                lower index
 *   topk_w        [T][k] float   softmax over the k selected logits
 *   topk_bits     [T][k] uint8   bit_table[token_req[t]][topk_idx[t][i]]
 *   hist          [E][L] int32   selection counts B_{j,k} (Sec. 3.4.3),
 *                                L = b_max-b_min+1, column = bit - b_min
 *   offsets       [E*L+1] int32  exclusive scan of hist (expert major)
 *   perm          [T*k] int32    slot ids t*k+i sorted stably by
 *                                (expert, bit): perm[position] = slot
 *   slot_of       [T*k] int32    inverse of perm: slot -> position
 *   expert_maxbit [E] uint8      largest requested bit-width, 0 if unused
 *   flags         [1] int32      bit 0: a table entry outside [b_min,b_max]
 *                                (clamped), bit 1: a token_req outside
 *                                [0,R) (clamped); 0 when all inputs valid
 */
typedef struct {
  float* logits;
  int32_t* topk_idx;
  float* topk_w;
  uint8_t* topk_bits;
  int32_t* hist;
  int32_t* offsets;
  int32_t* perm;
  int32_t* slot_of;
  uint8_t* expert_maxbit;
  int32_t* flags;
} d2moe_routing;

/*
 * Dual routing (Fig. 1, Sec. 3.2 bit-width per activated expert, Sec. 3.4
 * selection counts).  x: device [T][d] (x_dtype), Wg: device [E][d] float,
 * bias: device [E] float or NULL, token_req: device [T] int32 request id of
 * each token or NULL (all request 0), bit_table: device [R][E] uint8.
 * 1 <= k <= E <= 64, d >= 1, T >= 0.  The bit-width table stands in for the
 * paper's learned bit-width router, whose trained weights are not available.
 */
d2moe_status d2moe_route(const void* x, d2moe_dtype x_dtype, int32_t T,
                         int32_t d, const float* Wg, const float* bias,
                         int32_t E, int32_t k, const int32_t* token_req,
                         const uint8_t* bit_table, int32_t R, int32_t b_min,
                         int32_t b_max, const d2moe_routing* out,
                         void* stream);

/*
 * Dual routing with the learned bit-width routers of Sec. 3.2 in place of a
 * bit-width table: a lightweight router per expert scores the nest's
 * L = b_max - b_min + 1 candidate widths for each token (a softmax over those
 * scores gives the width probabilities the routers are trained with, Eq. 1),
 * and each activated expert runs at its router's most probable width.  The
 * router is read as one linear map per expert:
 *     bit_logits[t][e][l] = Wr[e][l] . x[t] + br[e][l],
 *     bits[t][i] = b_min + argmax_l bit_logits[t][topk_idx[t][i]][l]
 * (the lowest width wins ties).  Expert selection, weights, counts, scan and
 * permutation are exactly those of d2moe_route.
 *   Wr: device [E][L][d] float; br: device [E][L] float or NULL;
 *   bit_logits: device [T][E][L] float, written for every (token, expert).
 * Same constraints as d2moe_route (no request ids or table; flags stay 0).
 * The routers' trained weights are not available; callers supply their own.
 */
d2moe_status d2moe_route_learned(const void* x, d2moe_dtype x_dtype, int32_t T,
                                 int32_t d, const float* Wg, const float* bias,
                                 int32_t E, int32_t k, const float* Wr,
                                 const float* br, int32_t b_min, int32_t b_max,
                                 float* bit_logits, const d2moe_routing* out,
                                 void* stream);

/*
 * Workspace bytes needed by d2moe_moe_forward for these sizes (host): the
 * (expert, bit-width) work lists built from the counts B_{j,k} of Sec. 3.4.3,
 * the intermediate SwiGLU activations and expert outputs of the routed
 * (token, expert) pairs of Fig. 1, and the decode path's activation pieces.
 * shared_d_ff = 0 when there is no shared expert.
 */
d2moe_status d2moe_moe_forward_workspace(int32_t T, int32_t d, int32_t d_ff,
                                         int32_t E, int32_t k,
                                         int32_t shared_d_ff, size_t* bytes);

/*
 * MoE layer forward (Sec. 3.3.2 dequantization fused into the expert GEMMs):
 * for every routed (token, expert) pair at bit-width b,
 *     y = W2_b (silu(W1_b x) * (W3_b x)),
 *     out[t] = sum_i topk_w[t][i] * y(t, i)  [+ shared expert at shared_bits]
 * Each expert reads its planes only up to the bit-widths requested of it.
 *   x:    device [T][d] (x_dtype); out: device [T][d] (x_dtype)
 *   w13:  E experts of [2*d_ff][d] (W1 rows, then W3 rows)
 *   w2:   E experts of [d][d_ff]
 *   r:    routing produced by d2moe_route for the same T, E, k, ladder
 *         (uses topk_w, topk_bits, hist, offsets, perm, slot_of,
 *         expert_maxbit)
 *   shared_w13 / shared_w2: NULL, or 1 expert of [2*shared_d_ff][d] and
 *         [d][shared_d_ff], applied to every token with weight 1 at
 *         shared_bits (an always-on expert of fine-grained MoE layers)
 *   workspace: device buffer of at least d2moe_moe_forward_workspace bytes,
 *         256-byte aligned; contents need no initialisation.
 * Accumulation is fp32; bf16 outputs are rounded to nearest even.
 * Parts of the layer that do not depend on each other (the shared expert;
 * with more than 64 tokens, routed experts of at most 64 positions) run on
 * two side streams of the calling host thread, forked from `stream` and
 * joined back to it with events before the combine, so the call is ordered
 * on `stream` like any other and can be captured in a HIP graph from it.
 * The side streams and their events are created at the first such call of
 * a host thread on a device and kept until the process ends: make that
 * first call outside graph capture.
 */
d2moe_status d2moe_moe_forward(const void* x, d2moe_dtype x_dtype, int32_t T,
                               int32_t d, int32_t d_ff, int32_t E, int32_t k,
                               const d2moe_mwq* w13, const d2moe_mwq* w2,
                               const d2moe_routing* r,
                               const d2moe_mwq* shared_w13,
                               const d2moe_mwq* shared_w2,
                               int32_t shared_bits, int32_t shared_d_ff,
                               void* out, void* workspace, size_t ws_bytes,
                               void* stream);

/*
 * Same as d2moe_moe_forward, on `stream` alone (no side streams), and
 * additionally records events[0] / events[1]
 * (hipEvent_t) at the start / end of the W1-W3 expert kernel and events[2] /
 * events[3] at the start / end of the W2 expert kernel, on `stream`, so a
 * caller can time the expert kernels on the stream they run on.  Up to 64
 * tokens the events are the expert kernels' own start and end time stamps
 * (recorded as part of their launch, so timing adds no idle time to the
 * stream); above, they are recorded on the stream immediately before / after
 * the kernels.  events must hold four created events.  Nothing is recorded
 * when T == 0.
 */
d2moe_status d2moe_moe_forward_profiled(const void* x, d2moe_dtype x_dtype, int32_t T,
                                        int32_t d, int32_t d_ff, int32_t E, int32_t k,
                                        const d2moe_mwq* w13, const d2moe_mwq* w2,
                                        const d2moe_routing* r,
                                        const d2moe_mwq* shared_w13,
                                        const d2moe_mwq* shared_w2, int32_t shared_bits,
                                        int32_t shared_d_ff, void* out, void* workspace,
                                        size_t ws_bytes, void* stream,
                                        void* const* events);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * MoE layer forward as d2moe_moe_forward, with the workspace taken from a
 * fixed array of D2MOE_NOALLOC_SCRATCH_BYTES that the library holds on every
 * GPU it runs on (a static device array, kept until the process ends; its
 * address is looked up once per device at the first call on it).  The call
 * allocates nothing; the caller still owns x, the weights, the routing and
 * out, and everything runs on `stream` (no side streams are created).
 * Sizes whose workspace (d2moe_moe_forward_workspace) exceeds the
 * array return D2MOE_ESCRATCH before anything is launched: 32 MiB covers,
 * for example, decode of up to 64 tokens of the Mixtral-8x7B layer shape.
 * Every call on one GPU uses that GPU's one array, whatever the stream:
 * calls that overlap in time on the same GPU race on it and must be ordered
 * by the caller (one stream, or events).  The kernels need no initialised
 * workspace, so the array's contents left by a previous call do not matter.
 */
d2moe_status d2moe_moe_forward_noalloc(const void* x, d2moe_dtype x_dtype, int32_t T,
                                       int32_t d, int32_t d_ff, int32_t E, int32_t k,
                                       const d2moe_mwq* w13, const d2moe_mwq* w2,
                                       const d2moe_routing* r,
                                       const d2moe_mwq* shared_w13,
                                       const d2moe_mwq* shared_w2, int32_t shared_bits,
                                       int32_t shared_d_ff, void* out, void* stream);

/*
 * Residual update and normalisation between the MoE layers of a decoder
 * stack.  The decoders the paper evaluates (Mixtral-8x7B, LLaMA-MoE,
 * Sec. 5.1) feed every MoE layer the RMS-normalised hidden state and add the
 * layer's output to the residual stream; the normalisation weight is taken
 * as all ones:
 *     x[t] += y[t]                          (skipped when y is NULL)
 *     h[t]  = x[t] / sqrt(mean_c x[t][c]^2 + eps)
 *   x: device [T][d] float, the residual stream, updated in place
 *   y: device [T][d] (y_dtype, bf16 or f32) or NULL
 *   h: device [T][d] (h_dtype); bf16 is rounded to nearest even
 * 1 <= d <= 16384, T >= 0, eps >= 0.  Accumulation is fp32.
 */
d2moe_status d2moe_residual_rmsnorm(float* x, const void* y, d2moe_dtype y_dtype,
                                    int32_t T, int32_t d, float eps, void* h,
                                    d2moe_dtype h_dtype, void* stream);

/*
 * Bit-width-aware I/O-compute planning (Sec. 3.4), for weights streamed into
 * device memory rather than held there.
 *
 * One (expert, bit-width) unit of a layer: its computation is the `count`
 * requests routed to `expert` at `bits`; its load brings the expert's nested
 * planes (and their scales) from the width already on the device,
 * `load_from` (0: nothing), up to `load_to` (nothing when equal).
 */
typedef struct {
  int32_t expert, bits, load_from, load_to, count;
} d2moe_unit;

/*
 * Hottest-Expert-Bit-First order (Sec. 3.4.3): a queue per expert of its
 * requested bit-widths, ascending (so lower widths load first and are
 * reused, constraint 6b); repeatedly the queue head with the largest count
 * B_{j,k} (ties: the lower expert index) joins the I/O queue.  Host
 * function.  hist: host [E][L] selection counts (L = b_max - b_min + 1, as
 * d2moe_route writes them); resident: host [E] widths already on the device
 * or NULL (none); units: host array of at least E*L entries; *n_units
 * receives the count.
 */
d2moe_status d2moe_hebf_order(const int32_t* hist, int32_t E, int32_t b_min, int32_t b_max,
                              const uint8_t* resident, d2moe_unit* units, int32_t* n_units);

/* One step of a memory-budget plan: action 0 = free, 1 = load, of `level`
 * (0: base planes, scale and zero points; l >= 1: residual plane l and its
 * scales) of `expert` in `layer`. */
typedef struct {
  int32_t action, layer, expert, level;
} d2moe_budget_action;

/*
 * Memory-budget scheduler (Algorithm 2, Sec. 3.4.1) over one pass of
 * n_layers layers: for each layer, when the levels it still needs
 * (want[layer][expert] levels, 0 = unused) do not fit the budget left, the
 * levels of earlier layers are released, the previous layer first and its
 * highest levels first, the base level last, until they fit; then the
 * layer's missing levels are loaded.  Host function.
 *   level_bytes: host [K] bytes of one expert's level l;
 *   resident: host [n_layers][E] levels present, updated in place;
 *   actions: host array of max_actions entries; *n_actions the count
 *     (D2MOE_EINVAL, with *n_actions the count needed, if it is too small).
 * A layer that alone exceeds the budget is still loaded (the plan then
 * overdraws the budget; callers size the budget to at least one layer).
 */
d2moe_status d2moe_budget_plan(const uint8_t* want, int32_t n_layers, int32_t E,
                               const int64_t* level_bytes, int32_t K, int64_t budget,
                               uint8_t* resident, d2moe_budget_action* actions,
                               int32_t max_actions, int32_t* n_actions);

/*
 * The MoE layer forward with the expert weights streamed into device memory
 * (Sec. 3.4's bit-width-aware I/O-compute pipeline, for models whose
 * experts are not all resident): the units are executed in the given order
 * (e.g. from d2moe_hebf_order); each unit's nested delta is copied from the
 * host copy of the weights into the device copy on `io_stream`, and the
 * unit's bucket (its requests at its bit-width) is computed on `stream` as
 * soon as that copy has landed, so that the copy of a later unit overlaps
 * the computation of an earlier one (events[i] orders unit i).
 *   host_w13 / host_w2: the weights in host memory (pinned: allocated with
 *       hipHostMalloc), canonical layout, same shapes as w13 / w2;
 *   w13 / w2: the device copy (canonical layout) the kernels read;
 *   resident: host [E], the width each expert's planes already have in the
 *       device copy (0: none); updated to the widths after the call;
 *   hist_host: host [E][L], the routing's counts (copied from r->hist);
 *   units: must load each expert's planes in increasing width starting from
 *       `resident` and cover every nonempty bucket exactly once
 *       (D2MOE_EINVAL otherwise); events: n_units created hipEvent_t.
 * Other arguments as d2moe_moe_forward (no shared expert).  The per-token
 * arithmetic is that of d2moe_moe_forward's grouped-GEMM path (more than 64
 * tokens), whatever the batch.  Both streams are the caller's; the call
 * returns after enqueueing.
 */
d2moe_status d2moe_moe_forward_streamed(
    const void* x, d2moe_dtype x_dtype, int32_t T, int32_t d, int32_t d_ff, int32_t E, int32_t k,
    const d2moe_mwq* host_w13, const d2moe_mwq* host_w2, const d2moe_mwq* w13,
    const d2moe_mwq* w2, uint8_t* resident, const d2moe_routing* r, const int32_t* hist_host,
    const d2moe_unit* units, int32_t n_units, void* out, void* workspace, size_t ws_bytes,
    void* stream, void* io_stream, void* const* events);

/*
 * Measurement helper (not part of the layer): reads `bytes` of device memory
 * at `buf` once with 16-byte nontemporal loads in a grid-stride loop over
 * `blocks` workgroups of 256 threads and writes one XOR word per workgroup to
 * sink (device [blocks] uint32), so that the achieved HBM read rate of the
 * expert kernels can be set beside the rate a plain streaming read reaches
 * on the same GPU.  bytes % 16 == 0, buf 16-byte aligned, blocks >= 1.
 */
d2moe_status d2moe_stream_read(const void* buf, size_t bytes, uint32_t* sink, int32_t blocks,
                               void* stream);

#ifdef __cplusplus
}
#endif
#endif /* D2MOE_H */
