/*
 * stateflow.h -- C ABI of libstateflow, the MI355X (gfx950) hot path of
 * StateFlow's sequence-pipelined training for a gated linear recurrence layer.
 *
 * Operation (paper Sec. 2.1, Eq. 1, scalar-identity transition F_t = a_t I,
 * and the per-key-channel diagonal transition read for GLA; the state is
 * stored as S in R^{Dk x Dv}, the transpose of the paper's S):
 *
 *     S_t = a_t o S_{t-1} + k_t v_t^T,    o_t = S_t^T q_t,    a_t = exp(g_t)
 *
 * evaluated per (batch b, head h) in the chunkwise-parallel form of Sec. 2.2
 * (Eq. 2: Pre / ST / Out over kernel-level chunks of `chunk` tokens).  There is
 * no 1/sqrt(Dk) scaling (callers pre-scale q).  A segment ("chunk C_i" in
 * Sec. 3.1) enters with a boundary state S_in and leaves with S_out (Fwd
 * equation of Sec. 3.1); its backward consumes dS_out and produces dS_in (Bwd
 * equation of Sec. 3.1) for the loss  sum_t <dO_t, o_t> + <dS_out, S_out>.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Device pointers.  q, k, v, o, dO, dq, dk, dv, g, dg, states and the
 *    workspace are device (HBM) pointers on the current HIP device; the
 *    caller allocates and owns all of them.  The library never allocates or
 *    frees device memory and never synchronises the host; every call only
 *    enqueues work on the given stream(s) and returns.  Device faults surface
 *    at the caller's next synchronisation.
 *  - Layout.  q, k, dq, dk: [B][L][H][Dk];  v, o, dO, dv: [B][L][H][Dv], with
 *    element strides (sx_b, sx_l, sx_h) and the channel dim contiguous; all
 *    eight share the strides in sf_shape.  g, dg are float32: [B][L][H]
 *    (scalar gate, strides sg_b, sg_l, sg_h) or [B][L][H][Dk] (vector gate,
 *    channel dim contiguous).  g is the natural-log decay, dg its gradient.
 *    States (S_in, S_out, dS_out, dS_in, boundary slots) are float32
 *    [B][H][Dk][Dv], contiguous.
 *  - dtype.  io_dtype selects the element type of q, k, v, o, dO, dq, dk, dv:
 *    SF_F32 (fp32 arithmetic throughout, fp32 matrix cores) or SF_BF16
 *    (bf16 MFMA operands, fp32 accumulation and fp32 state).
 *  - Supported (v1): Dk == Dv in {64, 128}; chunk == 64 (0 selects 64);
 *    L % 64 == 0; SF_F32 with the per-channel gate needs Dk <= 64 (the scalar
 *    gate takes both head dims); pointers 16-byte aligned, strides a
 *    multiple of 16 bytes; 64 consecutive tokens of a tensor span < 2 GiB
 *    (63 * sx_l + Dk elements).  Anything else is rejected before any launch.
 *  - Errors.  Validation failures return a status synchronously and launch
 *    nothing.  A failed HIP call returns SF_E_HIP.  sf_last_error() gives a
 *    thread-local message for the last failure on the calling thread.  No C++
 *    exception crosses this boundary.
 *  - Aliasing.  No output may overlap any input or another output
 *    (SF_E_ALIAS).
 *  - Determinism.  Results are bitwise reproducible run to run and do not
 *    depend on the overlap mode.
 */
#ifndef STATEFLOW_H
#define STATEFLOW_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SF_ABI_VERSION 3

typedef enum {
    SF_OK = 0,
    SF_E_NULL = 1,        /* a required pointer is NULL */
    SF_E_SHAPE = 2,       /* inconsistent sizes or strides */
    SF_E_DTYPE = 3,       /* unknown io_dtype or gate kind */
    SF_E_ALIGN = 4,       /* pointer or stride not 16-byte aligned */
    SF_E_ALIAS = 5,       /* an output overlaps an input or another output */
    SF_E_WORKSPACE = 6,   /* workspace smaller than required */
    SF_E_UNSUPPORTED = 7, /* valid but not implemented in this version */
    SF_E_HIP = 8          /* a HIP runtime call failed */
} sf_status;

typedef enum { SF_F32 = 0, SF_BF16 = 1 } sf_dtype;
typedef enum { SF_GATE_SCALAR = 0, SF_GATE_VECTOR = 1 } sf_gate;

/* hipStream_t passed as an opaque pointer (NULL = the null stream). */
typedef void *sf_stream;

typedef struct sf_shape {
    int32_t B, H, Dk, Dv;
    int64_t L;        /* tokens: of the segment (segment calls) or of the whole
                         sequence (chain calls) */
    int32_t chunk;    /* kernel-level chunk length T_C (Sec. 2.2); 0 or 64 */
    int32_t io_dtype; /* sf_dtype */
    int32_t gate;     /* sf_gate */
    int32_t reserved; /* must be 0 */
    int64_t sx_b, sx_l, sx_h; /* element strides of the token tensors; all
                                 three 0 selects the packed [B][L][H][D] */
    int64_t sg_b, sg_l, sg_h; /* element strides of g / dg; all three 0
                                 selects the packed layout */
} sf_shape;

/*
 * Kernel timing for measurement, owned by the caller (no library state).
 * When sf_tuning.timing points at one of these, every launch of a kernel kind
 * k (an sf_kernel_id) with bit k of `mask` set takes the next free pair
 * (start[count], stop[count]) -- HIP events the caller created with timing
 * enabled -- as the begin and end timestamps of its own dispatch (no marker
 * packets are added to the stream), writes k to kind[count] and increments
 * count.  A launch that finds count == capacity increments `dropped` and is
 * not timed.  The library never creates, synchronises, reads or destroys the
 * events; the caller reads them after synchronising (hipEventElapsedTime).
 * One record must not be shared by calls running concurrently on several
 * host threads.
 */
typedef struct sf_timing {
    uint32_t mask;     /* bit k: time the launches of sf_kernel_id k */
    int32_t capacity;  /* pairs in start / stop / kind */
    int32_t count;     /* pairs used so far (the library increments it) */
    int32_t dropped;   /* timed launches that found no free pair */
    void **start;      /* hipEvent_t[capacity] */
    void **stop;       /* hipEvent_t[capacity] */
    int32_t *kind;     /* int32_t[capacity]: the kernel id of each used pair */
} sf_timing;

/* Kernel kinds: what one timed launch covers (sf_timing.mask bits). */
typedef enum {
    SF_K_FWD_PREP = 0,   /* per-superchunk state contribution (Pre) */
    SF_K_SCAN = 1,       /* fp32 state scan (ST / STB) */
    SF_K_FWD_OUT = 2,    /* intra-chunk attention + inter-chunk output (Out) */
    SF_K_BWD_PREP = 3,   /* per-superchunk state and state-gradient contributions */
    SF_K_BWD_DQ = 4,     /* dq by a forward state walk (OG) */
    SF_K_BWD_DKV = 5,    /* dk, dv, dg by a reverse state-gradient walk (PG) */
    SF_K_CONV_FWD = 6,   /* short convolution, forward */
    SF_K_CONV_BWD = 7,   /* short convolution, backward (dx, dtail_in, dw partials and their sum) */
    SF_K_GDN_PREP = 8,   /* gated delta rule: superchunk maps (M_J, N_J) */
    SF_K_GDN_SCAN = 9,   /* gated delta rule: fp32 affine state scan */
    SF_K_GDN_OUT = 10,   /* gated delta rule: output walk */
    SF_K_GDN_STORE = 11, /* gated delta rule backward: walk storing the state entering every chunk */
    SF_K_GDN_DPREP = 12, /* gated delta rule backward: superchunk state-gradient offsets E_J */
    SF_K_GDN_DSCAN = 13, /* gated delta rule backward: transposed scan */
    SF_K_GDN_DWALK = 14, /* gated delta rule backward: state-gradient walk */
    SF_K_GDN_DCHUNK = 15, /* gated delta rule backward: per-chunk parameter gradients */
    SF_K_COUNT = 16
} sf_kernel_id;

/* Tuning knobs; a NULL pointer selects the defaults for every field. */
typedef struct sf_tuning {
    int32_t ts;       /* state-materialisation stride in tokens (superchunk):
                         a multiple of 64, or 0 for automatic.  The state scan
                         (ST) runs over L/ts summaries per segment. */
    int32_t overlap;  /* chain calls: 1 (default when aux != NULL) runs the
                         state scans on the aux stream overlapped with the
                         neighbouring segment's dense kernels (Sec. 3.4
                         "Split and Overlap"); 2 (scalar and vector gate)
                         also moves each segment's preparation kernel to
                         aux, ahead of its scan, so that Pre and ST of one
                         segment run beside the output (or gradient)
                         kernels of its neighbour; 0 serialises on main.
                         Other values are rejected (SF_E_SHAPE); the delta
                         rule's chain treats 2 as 1. */
    int32_t reserved[4];
    sf_timing *timing; /* NULL: no timing (see sf_timing) */
} sf_tuning;

/* ABI version (SF_ABI_VERSION). */
int sf_abi_version(void);

/* Static text for a status code. */
const char *sf_status_str(int status);

/* Thread-local description of the most recent failure ("" if none). */
const char *sf_last_error(void);

/* Workspace bytes needed by sf_segment_fwd / sf_segment_bwd for this shape
 * (0 if the shape is invalid; the segment calls then report why). */
size_t sf_fwd_workspace_bytes(const sf_shape *shape, const sf_tuning *tuning);
size_t sf_bwd_workspace_bytes(const sf_shape *shape, const sf_tuning *tuning);

/*
 * One segment forward: (o, S_out) = Fwd(q, k, v, g; S_in)  (Sec. 3.1, Fwd).
 *   S_in   [B][H][Dk][Dv] f32, may be NULL (zero state, the paper's S_0 = 0).
 *   o      written for all L tokens; S_out written.
 *   ws     device scratch of at least sf_fwd_workspace_bytes(); contents on
 *          entry are ignored, on return unspecified.
 * L == 0 copies S_in (or zeros) to S_out.
 */
sf_status sf_segment_fwd(const sf_shape *shape, const void *q, const void *k, const void *v,
                         const float *g, const float *S_in, void *o, float *S_out, void *ws,
                         size_t ws_bytes, const sf_tuning *tuning, sf_stream stream);

/*
 * Allocation-free variant of sf_segment_fwd, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same operation, arguments, validation
 * and results as sf_segment_fwd with the same tuning (bitwise), but no
 * workspace argument: the superchunk states go to a scratch array that the
 * library holds in static device memory, SF_NOALLOC_SCRATCH_BYTES per GPU,
 * resident from the library's first use on that GPU until the process ends.
 * A shape whose workspace (sf_fwd_workspace_bytes) exceeds that size is
 * rejected with SF_E_WORKSPACE before any launch (a larger tuning.ts needs
 * less).  The call allocates nothing; the scratch's previous contents are
 * never read.  Every call on one GPU shares its scratch: calls that may run
 * concurrently on one GPU (other streams or host threads) race and must be
 * serialised by the caller.
 */
#define SF_NOALLOC_SCRATCH_BYTES (64u << 20)
sf_status sf_segment_fwd_noalloc(const sf_shape *shape, const void *q, const void *k, const void *v,
                                 const float *g, const float *S_in, void *o, float *S_out,
                                 const sf_tuning *tuning, sf_stream stream);

/*
 * One segment backward (Sec. 3.1, Bwd): given the forward inputs, S_in, the
 * output gradient dO and the boundary gradient dS_out (NULL = zero), writes
 * dq, dk, dv, dg and dS_in.  Nothing from the forward is reused: the states
 * are replayed from S_in (state replay "SR" of Sec. 3.4).
 */
sf_status sf_segment_bwd(const sf_shape *shape, const void *q, const void *k, const void *v,
                         const float *g, const float *S_in, const void *dO,
                         const float *dS_out, void *dq, void *dk, void *dv, float *dg,
                         float *dS_in, void *ws, size_t ws_bytes, const sf_tuning *tuning,
                         sf_stream stream);

/* Workspace bytes for the chain calls (covers both directions). */
size_t sf_chain_workspace_bytes(const sf_shape *shape, int32_t n_seg, const int64_t *seg_len,
                                const sf_tuning *tuning);

/*
 * Bytes of the kept superchunk states of a chain (optional `ckpt` buffer of
 * sf_chain_fwd / sf_chain_bwd): per segment of more than one superchunk, the
 * state entering each superchunk (the ST output of Sec. 2.2, fp32 Dk x Dv per
 * (b, h, superchunk)), each superchunk's log-decay and the state leaving the
 * segment.  The superchunk lengths are those the same shape, segments and
 * tuning select.  0 when no segment has more than one superchunk, and on
 * invalid arguments (then sf_last_error() is set).
 */
size_t sf_chain_ckpt_bytes(const sf_shape *shape, int32_t n_seg, const int64_t *seg_len,
                           const sf_tuning *tuning);

/*
 * Segment driver, forward (Sec. 3.1 chaining: S_0^in = S_init,
 * S_{i+1}^in = S_i^out).  shape->L is the whole sequence; seg_len[0..n_seg-1]
 * (host array, each > 0 and a multiple of 64) sums to it.  The token tensors
 * are the whole sequence; segment i covers tokens [sum_{j<i} seg_len[j], ...).
 *   S_bnd  [n_seg+1][B][H][Dk][Dv] f32: slot 0 is the input S_init (read);
 *          slots 1..n_seg receive S_out of each segment (slot n_seg = the
 *          final state).
 *   ckpt   NULL, or a device buffer of at least sf_chain_ckpt_bytes() bytes
 *          (16-byte aligned, caller-owned) that receives the superchunk
 *          states the forward computes anyway, so that sf_chain_bwd can read
 *          them instead of replaying the preparation and the forward scan.
 *          Its contents are only meaningful to sf_chain_bwd with the same
 *          shape, segments and tuning.
 * With aux != NULL and overlap enabled, each segment's state scan runs on aux
 * concurrently with the next segment's preparation and the previous
 * segment's output kernels (Sec. 3.4, fwd split-and-overlap schedule; with
 * overlap = 2 the preparation runs on aux too, ahead of the scan); both
 * streams must belong to the current device.  On return the work is
 * enqueued on main and aux, and main carries a dependency on all of it.
 */
sf_status sf_chain_fwd(const sf_shape *shape, int32_t n_seg, const int64_t *seg_len,
                       const void *q, const void *k, const void *v, const float *g, void *o,
                       float *S_bnd, void *ckpt, size_t ckpt_bytes, void *ws, size_t ws_bytes,
                       const sf_tuning *tuning, sf_stream main, sf_stream aux);

/*
 * Segment driver, backward (Sec. 3.1 reverse chaining dS_i^out = dS_{i+1}^in),
 * segments processed last to first.  S_bnd is the forward's boundary array
 * (slot i = S_in of segment i; slot n_seg is not read).  dS_final is the
 * gradient of the final state (NULL = zero); dS_init receives the gradient
 * of S_init.  Overlap as in sf_chain_fwd (Sec. 3.4, bwd schedule).
 * ckpt: NULL (every superchunk state is recomputed: the preparation replays
 * D_J and the scan runs forward again), or the buffer that sf_chain_fwd
 * filled for the same shape, segments and tuning (read only; at least
 * sf_chain_ckpt_bytes() bytes).  The results are the same either way.
 */
sf_status sf_chain_bwd(const sf_shape *shape, int32_t n_seg, const int64_t *seg_len,
                       const void *q, const void *k, const void *v, const float *g,
                       const float *S_bnd, const void *ckpt, size_t ckpt_bytes, const void *dO,
                       const float *dS_final, void *dq, void *dk, void *dv, float *dg,
                       float *dS_init, void *ws, size_t ws_bytes, const sf_tuning *tuning,
                       sf_stream main, sf_stream aux);

/*
 * Short convolution with a boundary tail: the auxiliary boundary state that
 * Sec. 3.1 (footnote to the chunk boundary states) lets a segment carry next
 * to S.  Per batch b, channel c and token t of a segment, with a causal
 * depthwise window of W taps:
 *
 *     u_t[c] = sum_{j=0}^{W-1} w[c][j] * xh_{t-W+1+j}[c],     y_t[c] = act(u_t[c])
 *
 * where xh_s = x_s for s >= 0 and xh_s = tail_in[b][W-1+s][c] for
 * -(W-1) <= s < 0: the last W-1 inputs of the previous segment, oldest first
 * (NULL = zeros, the start of a sequence).  tail_out[b][i][c] = xh_{L-W+1+i}
 * (i = 0..W-2) is the tail the next segment takes, so chaining segments
 * through their tails equals one call over the whole sequence.
 *   x, y, dx, dy   [B][L][C] in io_dtype, element strides (sx_b, sx_l),
 *                  channels contiguous (0, 0 = packed)
 *   w, dw          [C][W] float32
 *   tail_in, tail_out, dtail_in, dtail_out   [B][W-1][C] float32, packed
 *   act            SF_ACT_NONE (identity) or SF_ACT_SILU (u * sigmoid(u))
 * The backward takes the gradient of the loss sum <dy, y> + <dtail_out,
 * tail_out> (dtail_out NULL = zero) and writes dx, dtail_in and dw (summed
 * over batch and tokens, in a fixed order: bitwise reproducible).  dw needs
 * a workspace of sf_conv_bwd_workspace_bytes().  Supported: 1 <= W <= 4
 * (W = 1 has no tail; the tail pointers are then ignored), C a multiple of 8,
 * L >= 0, 16-byte aligned pointers and strides.  tuning may be NULL; of its
 * fields only `timing` applies here.  Same ownership, error and aliasing rules
 * as the recurrence entry points.
 */
typedef enum { SF_ACT_NONE = 0, SF_ACT_SILU = 1 } sf_act;

typedef struct sf_conv_shape {
    int32_t B, C;     /* batch, channels */
    int64_t L;        /* tokens of the segment */
    int32_t W;        /* taps, 1..4 */
    int32_t io_dtype; /* sf_dtype of x, y, dx, dy */
    int32_t act;      /* sf_act */
    int32_t reserved; /* must be 0 */
    int64_t sx_b, sx_l; /* element strides of x, y, dx, dy; both 0 = packed */
} sf_conv_shape;

size_t sf_conv_bwd_workspace_bytes(const sf_conv_shape *shape);
sf_status sf_conv_fwd(const sf_conv_shape *shape, const void *x, const float *w, const float *tail_in,
                      void *y, float *tail_out, const sf_tuning *tuning, sf_stream stream);
sf_status sf_conv_bwd(const sf_conv_shape *shape, const void *x, const float *w, const float *tail_in,
                      const void *dy, const float *dtail_out, void *dx, float *dw, float *dtail_in,
                      void *ws, size_t ws_bytes, const sf_tuning *tuning, sf_stream stream);

/*
 * Hybrid-aware segment lengths (Sec. 3.2, Hybrid-Aware Sequence Chunking):
 * host-only, no device work.  For a sequence of T tokens cut into N segments
 * with boundaries 0 = c_0 < c_1 < ... < c_N = T, the paper prices segment i at
 *     Cost_i = w_tok * s_i + w_soft * (c_i * s_i + s_i^2 / 2),   s_i = c_{i+1} - c_i,
 * where w_tok = L_lin * C_lin + C_dense (per-token FLOPs of the linear
 * recurrence layers and the dense work) and w_soft = L_soft * C_soft (FLOPs
 * per query-key pair of the softmax layers).  The balanced boundaries
 * c_i^hybrid make every Cost_i equal; the candidates are
 *     c_i(alpha) = (1 - alpha) * i * T / N + alpha * c_i^hybrid,
 * each rounded to the closest multiple of `round_to` (half-way cases round
 * up).  seg_len[0..N-1] receives c_{i+1} - c_i.
 *   T > 0 and a multiple of round_to; N >= 1; round_to >= 1; alpha >= 0;
 *   w_tok >= 0, w_soft >= 0, not both 0.
 * SF_E_SHAPE if an argument is out of range or rounding leaves a segment
 * empty; SF_E_NULL if seg_len is NULL.
 */
sf_status sf_partition_hybrid(int64_t T, int32_t N, double alpha, double w_tok, double w_soft, int32_t round_to,
                              int64_t *seg_len);

/*
 * Gated delta rule (Gated DeltaNet, the scalar-plus-low-rank transition of
 * Sec. 2.1), forward over one segment:
 *     S_t = a_t (I - beta_t k_t k_t^T) S_{t-1} + beta_t k_t v_t^T,   o_t = S_t^T q_t,
 * a_t = exp(g_t), S stored as [Dk][Dv] (the transpose of the paper's S).
 * q, k, v, o as for sf_segment_fwd (shape->io_dtype must be SF_BF16,
 * Dk == Dv in {64, 128}, scalar gate, L a multiple of 64); g and beta are
 * float32 [B][L][H] with the gate strides of `shape`; S_in may be NULL (zero
 * state); S_out receives the final state; v_new, if not NULL, receives the
 * corrected values u_t = beta_t (v_t - a_t S_{t-1}^T k_t) (the V^new that the
 * delta rule's ST step returns beside the state, Sec. 2.1), bf16 with the
 * layout of v.
 * Superchunks of tuning->ts tokens (0: chosen from the shape and the device's
 * CU count) run in parallel: since one chunk's update is affine in the state,
 * each superchunk J reduces to S_{J+1} = M_J S_J + N_J (dense M_J, N_J,
 * Sec. 2.2's Pre step with a matrix-valued transition), an fp32 scan over J
 * gives every S_J (ST), and the output walk runs from them (Out).
 *   ws  device scratch of at least sf_gdn_fwd_workspace_bytes() (0 when the
 *       segment is one superchunk); contents on entry ignored, on return
 *       unspecified.
 * Same ownership, validation, aliasing and error rules as the other entry
 * points.
 */
size_t sf_gdn_fwd_workspace_bytes(const sf_shape *shape, const sf_tuning *tuning);
sf_status sf_gdn_fwd(const sf_shape *shape, const void *q, const void *k, const void *v, const float *g,
                     const float *beta, const float *S_in, void *o, float *S_out, void *v_new, void *ws,
                     size_t ws_bytes, const sf_tuning *tuning, sf_stream stream);

/*
 * Gated delta rule backward over one segment: given the forward's inputs,
 * S_in (NULL: zero), dO and dS_out (NULL: zero), the gradients of
 *     Loss = sum_t <dO_t, o_t> + <dS_out, S_out>
 * with respect to q, k, v (bf16, layout of q), g and beta (float32, layout of
 * g) and S_in (dS_in, float32 [B][H][Dk][Dv]; written also when S_in is NULL).
 * The states are recomputed (superchunk prep, fp32 scan, and a walk that
 * stores the state entering every chunk); the state gradient runs backwards
 * over the chunks (dS_start = M_J^T dS_end + E_J per superchunk, the
 * transpose of the forward's chunk map) and is stored for every chunk; the
 * parameter gradients of all chunks are then computed in parallel.
 *   ws  device scratch of at least sf_gdn_bwd_workspace_bytes(): two fp32
 *       D x D states per 64-token chunk plus the superchunk maps; contents
 *       on entry ignored.
 * Same shape rules as sf_gdn_fwd; same ownership, validation, aliasing and
 * error rules as the other entry points.
 */
size_t sf_gdn_bwd_workspace_bytes(const sf_shape *shape, const sf_tuning *tuning);
sf_status sf_gdn_bwd(const sf_shape *shape, const void *q, const void *k, const void *v, const float *g,
                     const float *beta, const float *S_in, const void *dO, const float *dS_out, void *dq, void *dk,
                     void *dv, float *dg, float *dbeta, float *dS_in, void *ws, size_t ws_bytes,
                     const sf_tuning *tuning, sf_stream stream);

/*
 * Gated delta rule over n_seg consecutive segments (Sec. 3.1 chaining), one
 * call each way.  Shapes and per-token tensors as for sf_gdn_fwd with
 * shape->L = sum of seg_len (each a positive multiple of 64).
 *   S_bnd  [n_seg + 1][B][H][Dk][Dv] f32: slot 0 is S_init (input, zeros for
 *          a zero state); the forward writes slot i+1 = the state after
 *          segment i.  The backward reads slots 0 .. n_seg-1.
 *   v_new  optional (NULL to skip), as for sf_gdn_fwd.
 *   dS_final  optional gradient of the state after the last segment.
 *   dS_init   receives the gradient of S_init.
 *   ws     at least sf_gdn_chain_workspace_bytes(); contents on entry ignored.
 *   ckpt   NULL, or a caller buffer (16-byte aligned) of at least
 *          sf_gdn_chain_ckpt_bytes(): the forward writes there, per segment of
 *          more than one superchunk, the state entering every superchunk and
 *          every superchunk's map M_J (fp32 Dk x Dk); the backward, given the
 *          buffer the forward filled for the same shape, segments and tuning,
 *          reads them instead of running the prep walk and the state scan
 *          again.  The results are the same either way.
 * With aux != NULL (and tuning->overlap != 0) the state scans run on aux:
 * forward, the scan of each segment (which then also writes S_bnd[i+1]) runs
 * alongside the previous segment's output walk; backward, the state scan
 * alongside the dS prep and the dS scan alongside the state-storing walk
 * (Sec. 3.4, "Split and Overlap").  Results do not depend on the overlap.
 * Both streams must belong to the current device; on return, work is queued on
 * main that waits for everything queued on aux.
 */
size_t sf_gdn_chain_workspace_bytes(const sf_shape *shape, int32_t n_seg, const int64_t *seg_len,
                                    const sf_tuning *tuning);
/* Bytes of the kept states and maps (0 when no segment has more than one
 * superchunk, and on invalid arguments, with sf_last_error() set). */
size_t sf_gdn_chain_ckpt_bytes(const sf_shape *shape, int32_t n_seg, const int64_t *seg_len,
                               const sf_tuning *tuning);
sf_status sf_gdn_chain_fwd(const sf_shape *shape, int32_t n_seg, const int64_t *seg_len, const void *q,
                           const void *k, const void *v, const float *g, const float *beta, void *o, float *S_bnd,
                           void *ckpt, size_t ckpt_bytes, void *v_new, void *ws, size_t ws_bytes,
                           const sf_tuning *tuning, sf_stream main, sf_stream aux);
sf_status sf_gdn_chain_bwd(const sf_shape *shape, int32_t n_seg, const int64_t *seg_len, const void *q,
                           const void *k, const void *v, const float *g, const float *beta, const float *S_bnd,
                           const void *ckpt, size_t ckpt_bytes, const void *dO, const float *dS_final, void *dq,
                           void *dk, void *dv, float *dg, float *dbeta, float *dS_init, void *ws, size_t ws_bytes,
                           const sf_tuning *tuning, sf_stream main, sf_stream aux);


#ifdef __cplusplus
}
#endif
#endif /* STATEFLOW_H */
