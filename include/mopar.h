/*
 * mopar.h -- C ABI of the MI355X (gfx950) sliced-inference library.
 *
 * The library implements the hot path of MOPAR (arXiv 2404.02445): a model
 * cut vertically into slices of similar layers (Sec. III-C, strategy pi_S),
 * each resource-dominant (RD) conv / GEMM split into k equal-size sub-slices
 * along its output channels or features (Sec. III-C, strategy pi_P), and the
 * activation at every split point handed to the next slice through a device
 * buffer, optionally encoded by the one-layer autoencoder of Sec. III-D.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Status.    Every call returns a mopar_status.  On any non-zero status
 *            nothing has been enqueued and no output has been written;
 *            mopar_last_error() returns a description (thread-local).
 * Memory.    The caller owns every byte: weights, inputs, outputs, code
 *            buffers and the workspace are device pointers the caller
 *            allocated; descriptors and plans are host memory the caller
 *            owns.  The library never allocates device memory, never frees
 *            caller memory and never synchronises the host -- except
 *            mopar_model_measure and mopar_model_op_times, which wait for
 *            their timing events, as documented there.
 * Streams.   `stream` is a hipStream_t passed as void* (NULL = the default
 *            stream).  Work is enqueued asynchronously in call order.
 * Alignment. Device pointers must be 16-byte aligned.
 * Sizes.     Every GEMM operand -- an op's input activation (for a conv, the
 *            whole input image batch), its weight matrix, a boundary tensor
 *            and its code -- must stay under 2 GiB; a model or codec that
 *            needs more is rejected with MOPAR_E_UNSUPPORTED before anything
 *            is enqueued.
 * Layouts.   Tensor descriptors give logical dims in canonical order:
 *            images (N, C, H, W), flattened (N, F), sequences (B, S, F),
 *            token ids (B, S).  Physically, the model input is stored as
 *            described (images: NCHW float32; ids: int32), and every other
 *            rank-4 tensor is stored channels-last (NHWC) in the model
 *            dtype; rank-2/3 tensors are row-major.  Weight layouts are
 *            given at mopar_op.
 * Determinism. Plans and sub-slice ranges are pure functions of their
 *            inputs, and a forward pass is bitwise reproducible: no kernel
 *            accumulates through atomics.  Two kernels hand out work with
 *            atomics -- the one-launch LSTM recurrence, whose blocks claim
 *            (step, tile) work, and the persistent GEMM, whose blocks take
 *            tiles from a counter -- and both compute a tile with the same
 *            operands and operation order whichever block takes it.  The k-way
 *            sub-sliced RD kernels produce the same bits as the unsplit
 *            kernel.
 */
#ifndef MOPAR_H
#define MOPAR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MOPAR_OK = 0,
    MOPAR_E_ARG = 1,          /* null pointer, bad enum, inconsistent sizes        */
    MOPAR_E_SHAPE = 2,        /* tensor shapes do not match the op                 */
    MOPAR_E_DTYPE = 3,        /* dtype not supported for this op / model           */
    MOPAR_E_UNSUPPORTED = 4,  /* valid request outside what the kernels implement  */
    MOPAR_E_INFEASIBLE = 5,   /* no plan satisfies the slicing constraints         */
    MOPAR_E_WORKSPACE = 6,    /* workspace or code buffer too small                */
    MOPAR_E_HIP = 7           /* a HIP runtime call or kernel launch failed        */
} mopar_status;

typedef enum { MOPAR_F32 = 0, MOPAR_BF16 = 1, MOPAR_I32 = 2 } mopar_dtype;

/* ------------------------------------------------------------------------ */
/* Sub-slice ranges (Sec. III-C: eta equal-size sub-slices)                  */
/* ------------------------------------------------------------------------ */

/* Range [*lo, *hi) of sub-slice j when n outputs are split k ways: sizes
 * n/k, with the first n mod k ranges one larger.  Needs 1 <= k <= n,
 * 0 <= j < k; otherwise MOPAR_E_ARG. */
int mopar_subslice_range(int32_t n, int32_t k, int32_t j, int32_t* lo, int32_t* hi);

/* ------------------------------------------------------------------------ */
/* Planning (Sec. III-B service profile, Sec. III-C HyPAD, Eq. 1-6, Alg. 1)  */
/* ------------------------------------------------------------------------ */

/* One planning node (layer): memory footprint M_l (bytes) and time t_l
 * (seconds) of Eq. 1-3, the bytes of the tensor it hands to the next node,
 * and the output width of its RD op(s) (smallest one; 0 = no RD op). */
typedef struct {
    double mem_bytes;
    double time_s;
    double out_bytes;
    int32_t rd_width;
    int32_t reserved;
} mopar_layer_profile;

/* Options of the partitioner; zero-initialise and set what you need. */
typedef struct {
    int32_t n_slices;           /* 0: the DP picks the count; > 0: exactly this many slices       */
    int32_t k_max;              /* largest sub-slice count searched (>= 1; 0 is read as 1)        */
    const uint8_t* allowed_cut; /* n-1 flags, cut after node j allowed; NULL: all, after node
                                   elimination; when given, elimination is skipped               */
    double elim_tau;            /* node-elimination threshold (Sec. III-C: 0.05); < 0 disables    */
    double c_m;                 /* cost per unit memory x time (Eq. 6)                            */
    double c_n;                 /* cost per unit transfer time (Eq. 6)                            */
    double bw_Bps;              /* boundary bandwidth for t_c = (bytes / ratio) / bw (> 0)        */
    const double* ratio;        /* n-1 compression ratios per cut position; NULL: 1               */
    double lambda_bytes;        /* eta <= floor(M_g / lambda) when > 0 (Eq. 6 constraint)         */
    const double* tp_table;     /* [n][k_max] measured t_p(l, eta); NULL: t_p = t_l               */
    const double* ta_table;     /* [n][k_max] measured t_a(l, eta); NULL: 0                       */
    const int32_t* k_override;  /* n entries; > 0 forces k for that node (at most the node's RD
                                   width, and at most k_max when measured tables are given); NULL: none */
    int32_t uniform;            /* 1: the Uniform partitioning of the evaluation (Sec. IV): exactly
                                   n_slices (> 0) slices with equal node counts (the first
                                   n mod n_slices one node longer); allowed_cut and elimination do
                                   not apply; the parallelism search, cost and latency as usual   */
    int32_t reserved;
} mopar_plan_opts;

/* A plan.  slice_end and k are caller-allocated arrays of n entries. */
typedef struct {
    int32_t n_layers;           /* n: set by the caller to the array capacity; checked            */
    int32_t n_slices;           /* out                                                            */
    int32_t* slice_end;         /* out: last node (0-based) of each slice                         */
    int32_t* k;                 /* out: sub-slice count per node (1 = unsplit)                    */
    double cost;                /* out: Eq. 6 objective of the chosen cuts                        */
    double t_tau;               /* out: Eq. 5 latency with the chosen k and cuts                  */
    double t_unsplit;           /* out: sum of t_l                                                */
    int32_t latency_ok;         /* out: t_tau <= t_unsplit (Eq. 6, second constraint)             */
    int32_t reserved;
} mopar_plan;

/* HyPAD on a chain of n planning nodes (Alg. 1): node elimination, DP over
 * split points (ties keep the longest last slice), backtrack through the
 * stored argmin, then the parallelism search per slice (Eq. 5; ties keep
 * the smallest eta).  Pure host code, no device calls.  Errors: MOPAR_E_ARG
 * (null pointers, n < 1, capacity too small, bad k_override),
 * MOPAR_E_INFEASIBLE (fewer admissible cuts than n_slices - 1). */
int mopar_plan_slices(const mopar_layer_profile* layers, int32_t n, const mopar_plan_opts* opts,
                      mopar_plan* out);

/* ------------------------------------------------------------------------ */
/* Model description                                                         */
/* ------------------------------------------------------------------------ */

typedef struct {
    int32_t dtype;              /* mopar_dtype */
    int32_t rank;               /* 1..4 */
    int64_t dims[4];            /* canonical order, see the header comment */
} mopar_tensor_desc;

typedef enum {
    MOPAR_OP_CONV = 1,       /* in0 (N,C,H,W) -> out (N,Co,Ho,Wo); in1 optional residual (out shape)
                                w: [Co][kh][kw][Cs] with Cs = C rounded up to the kernel's channel
                                granule (8 for bf16, 4 for f32; extra channels zero); b: [Co]
                                When in0 is the model input (NCHW float32) the library converts it
                                to channels-last itself.                                          */
    MOPAR_OP_LINEAR = 2,     /* in0 (..., K) or (N,C,H,W) flattened -> out (..., n_out);
                                in1 optional residual; w: [n_out][K] (for an image input, K runs
                                over (h, w, c) -- channels-last order); b: [n_out]                */
    MOPAR_OP_MAXPOOL = 3,    /* kh x kw window, stride, pad (outside = -inf)                      */
    MOPAR_OP_AVGPOOL = 4,    /* global average (N,C,H,W) -> (N,C)                                 */
    MOPAR_OP_LAYERNORM = 5,  /* over the last dim of in0 (+ in1); w: gamma [F]; b: beta [F]; eps   */
    MOPAR_OP_ATTENTION = 6,  /* in0 (B,S,3F) = [Q|K|V] -> out (B,S,F); heads; scale; head dim 64  */
    MOPAR_OP_EMBED_BERT = 7, /* ids (B,S) -> LN(tok[id] + pos[s] + type[0]); w: tok [V][F];
                                w2: pos [P][F]; w3: type [T][F]; w4: gamma; w5: beta; eps        */
    MOPAR_OP_EMBED = 8,      /* ids (B,S) -> table[id]; w: table [V][F].  For both embeddings an
                                id outside [0, V) is clamped to the nearest row (no error, no
                                access past the table); V < 2^31                                 */
    MOPAR_OP_LSTM = 9        /* in0 (B,T,E) -> out (B,T,H) hidden sequence, h0 = c0 = 0;
                                w: W_ih [4H][E], w2: W_hh [4H][H], b: b_ih [4H], w3: b_hh [4H];
                                rows interleaved by unit: row 4u+g holds gate g (i,f,g,o) of
                                hidden unit u.  c is kept in float32.                              */
} mopar_op_kind;

typedef enum { MOPAR_ACT_NONE = 0, MOPAR_ACT_RELU = 1, MOPAR_ACT_GELU = 2 } mopar_act;

/* One operator.  Weight fields are byte offsets into the weight blob passed
 * to mopar_model_create (-1 = absent); weights are in the model dtype. */
typedef struct {
    int32_t kind;               /* mopar_op_kind */
    int32_t act;                /* mopar_act (conv, linear) */
    int32_t layer;              /* planning node, non-decreasing over the op list */
    int32_t branch;             /* 0: sequential chain (Eq. 1); >= 1: parallel branch (Eq. 2) */
    int32_t pos;                /* position along its branch (Eq. 2) */
    int32_t rd;                 /* 1: resource-dominant, split k ways as the plan says */
    int32_t in0, in1, out;      /* tensor ids; in1 = -1 when absent */
    int32_t kh, kw, stride, pad;
    int32_t heads;
    int32_t n_out;              /* conv C_out, linear N, LSTM hidden size */
    int32_t out_off;            /* conv: first channel of `out` this op writes.  When out has more
                                   channels than n_out, the op fills channels [out_off,
                                   out_off + n_out) -- the branches of a parallel node concatenated
                                   in place (Sec. III-B, parallel topology); the writers of one
                                   tensor sit in one node, tile its channels exactly, take no
                                   residual, and precede every reader.  0 otherwise. */
    float eps;
    float scale;
    int64_t rows[3];            /* table rows: EMBED_BERT vocab, positions, token types; EMBED vocab */
    int64_t w, b, w2, w3, w4, w5;
} mopar_op;

typedef struct {
    int32_t dtype;              /* model dtype: MOPAR_F32 or MOPAR_BF16 */
    int32_t n_tensors;
    const mopar_tensor_desc* tensors;
    int32_t n_ops;
    const mopar_op* ops;
    int32_t n_layers;
    int32_t input, output;      /* tensor ids of the model input and output */
} mopar_model_desc;

typedef struct mopar_model_s* mopar_model_t;

/* Validate the description and build host metadata: the graph G = <V, E> of
 * operators grouped into planning nodes (layers) with single-input topology,
 * each node's ops in the chain / parallel-branch structure that Eq. 1-3
 * aggregate, the resource-dominant ops that the hybrid strategy pi_P may split
 * (Sec. III-B service profile, Sec. III-C problem statement), and the
 * workspace layout.  `weights_dev` (device) must stay valid for the model's
 * life; `weights_bytes` bounds every weight offset.  No device calls.
 * Errors: MOPAR_E_ARG (null pointers, bad ids or offsets, a graph the planner
 * cannot chain), MOPAR_E_SHAPE, MOPAR_E_DTYPE, MOPAR_E_UNSUPPORTED (a valid
 * model outside what the kernels implement); *out is NULL then. */
int mopar_model_create(const mopar_model_desc* desc, const void* weights_dev, size_t weights_bytes,
                       mopar_model_t* out);
void mopar_model_destroy(mopar_model_t model);

/* Layer profiles (Eq. 1-4) of the model: op memory = bytes of parameters +
 * inputs + output; op time = max(FLOP / peak, bytes / 8e12), peak 2.5e15
 * (bf16) or 157.3e12 (f32) FLOP/s; FLOP counted for conv, linear, attention
 * and LSTM.  out_bytes of node j < n_layers - 1 is the size of every tensor
 * crossing the cut after it (mopar_model_cut_tensors), of the last node its
 * output.  `out` has n_layers entries. */
int mopar_model_profile(mopar_model_t model, mopar_layer_profile* out);

/* The same profile built from each node's dominant operators only (Sec.
 * III-B): the node's ops sorted by memory footprint, largest first (ties by
 * position), and the shortest such prefix whose footprint reaches `frac`
 * (the paper: 0.8) of the node's total, the total summed in op order and the
 * prefix in sorted order.  Eq. 1-3 then aggregate the selected ops; out_bytes
 * and rd_width are those of the whole node.  frac must be in (0, 1]. */
int mopar_model_profile_dominant(mopar_model_t model, double frac, mopar_layer_profile* out);

/* Bytes of device workspace mopar_slice_forward / mopar_model_forward need
 * under `plan`: the tensors that live inside slices, the boundary tensors
 * before encode and after decode (the hand-off of Sec. III-D goes through the
 * caller's code buffers, not this workspace) and op scratch (split-K partial
 * sums, the LSTM gate pre-activations and cell state, the tile counters of a
 * persistent GEMM launch).  The caller allocates it
 * (Memory convention); one workspace serves one forward at a time.  Errors:
 * MOPAR_E_ARG (null pointers, a plan for another model or with an invalid k). */
int mopar_model_workspace_bytes(mopar_model_t model, const mopar_plan* plan, size_t* bytes);

/* Run slice s of `plan`: one slice of the vertical partition pi_S (Sec.
 * III-C; the paper deploys each slice as its own function), i.e. the layers
 * after the previous split point up to slice_end[s].  `in_dev` holds the slice
 * input (the model input for s = 0, otherwise the output of node
 * slice_end[s-1], in its physical layout); `out_dev` receives the output of
 * node slice_end[s].  Any other tensor crossing the cut before slice s (a skip
 * edge, see mopar_model_cut_tensors) is read from its slot in `ws`, where the
 * earlier slices, run with the same workspace, left it.  RD ops of node l run
 * as the k[l] equal-size sub-slices of pi_P, all in one launch, each writing
 * its own output columns (the aggregation t_a of Eq. 5 costs nothing).
 * Errors: MOPAR_E_ARG (bad plan, s out of range, null pointers),
 * MOPAR_E_WORKSPACE (ws smaller than mopar_model_workspace_bytes), MOPAR_E_HIP. */
int mopar_slice_forward(mopar_model_t model, const mopar_plan* plan, int32_t s, const void* in_dev,
                        void* out_dev, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Boundary codec (Sec. III-D)                                               */
/* ------------------------------------------------------------------------ */

typedef enum { MOPAR_CODEC_RAW = 0, MOPAR_CODEC_AE = 1 } mopar_codec_kind;

/* RAW: the code is the tensor's bytes (lossless, R = 1).
 * AE:  at every position p (each (n,h,w) of an image, each token of a
 *      sequence): code[p][e] = b_enc[e] + sum_c w_enc[e][c] x[p][c] and
 *      y[p][c] = b_dec[c] + sum_e w_dec[c][e] code[p][e], stored in the
 *      tensor's dtype; R = c / c_code.  Weights are device pointers in the
 *      tensor dtype: w_enc [c_code][c], b_enc [c_code], w_dec [c][c_code],
 *      b_dec [c].  Any c, c_code >= 1: a layer whose input width (c for the
 *      encoder, c_code for the decoder) is a multiple of 8 (bf16) or 4 (f32)
 *      runs on the matrix cores, any other on the vector ALUs (such layers are
 *      a few channels wide).  positions * max(c, c_code) < 2^31. */
typedef struct {
    int32_t kind;
    int32_t c, c_code;
    int32_t reserved;
    const void* w_enc;
    const void* b_enc;
    const void* w_dec;
    const void* b_dec;
} mopar_codec;

/* Size in bytes of the code of tensor x. */
int mopar_boundary_code_bytes(const mopar_codec* codec, const mopar_tensor_desc* x, size_t* bytes);

/* Encode x (device, physical layout) into code_dev.  Channels are dims[1]
 * for rank-4 tensors and the last dim otherwise. */
int mopar_boundary_encode(const mopar_codec* codec, const mopar_tensor_desc* x, const void* x_dev,
                          void* code_dev, void* stream);

/* Decode code_dev into y (device), the inverse direction of encode. */
int mopar_boundary_decode(const mopar_codec* codec, const mopar_tensor_desc* y, const void* code_dev,
                          void* y_dev, void* stream);

/* ------------------------------------------------------------------------ */
/* Whole model                                                               */
/* ------------------------------------------------------------------------ */

/* Sliced forward pass: for each slice s, decode the tensors crossing the cut
 * before it (s > 0), run the slice, and encode the tensors crossing the cut
 * after it (s < S-1), all on `stream` with no host round-trip (the device
 * buffers and stream order stand for the share-memory directory and message
 * channel of Sec. III-D).  A cut after node j carries the tensors of
 * mopar_model_cut_tensors(j): one for a chain of single-input nodes, more
 * where skip edges cross it.  `codecs` and `code_bufs` have one entry per
 * boundary tensor -- the tensors of cut 0 in ascending id, then those of
 * cut 1, ... (S-1 entries for a chain; may be NULL when S = 1); each buffer
 * holds mopar_boundary_code_bytes of its tensor. */
int mopar_model_forward(mopar_model_t model, const mopar_plan* plan, const mopar_codec* codecs,
                        const void* in_dev, void* out_dev, void* const* code_bufs, void* ws,
                        size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory -- code under HIP graph
 * capture, serving loops or harnesses that forbid hipMalloc: mopar_model_forward
 * with the workspace taken from a static device array the library owns
 * (MOPAR_STATIC_WORKSPACE_BYTES per GPU, held until the process ends) instead of
 * a caller buffer.  Inputs, outputs and code buffers are still the caller's.
 * The call allocates nothing (its first call on a GPU looks the array's device
 * address up once).  Same kernels, hence the same output bits, as
 * mopar_model_forward.  Every call on one GPU shares that GPU's array: calls
 * that overlap on one GPU (other streams, other threads) race and must be
 * ordered by the caller.  The forward writes every workspace byte it reads, so
 * the array's contents from an earlier call do not matter.
 * Errors: as mopar_model_forward; MOPAR_E_WORKSPACE when the plan needs more
 * than MOPAR_STATIC_WORKSPACE_BYTES (mopar_model_workspace_bytes tells), before
 * any device call; MOPAR_E_ARG while per-op timing is on (it creates events). */
#define MOPAR_STATIC_WORKSPACE_BYTES ((size_t)64 << 20)
int mopar_model_forward_static(mopar_model_t model, const mopar_plan* plan, const mopar_codec* codecs,
                               const void* in_dev, void* out_dev, void* const* code_bufs, void* stream);

/* The tensors a cut after node `node` (0 <= node < n_layers - 1) carries: the
 * outputs of nodes <= node that nodes > node read (Sec. III-C: after node
 * elimination, the parallel edges between the two sides are one merged edge
 * whose size is their sum -- mopar_model_profile's out_bytes of that node).
 * Writes up to `cap` tensor ids in ascending order to tids; *count = all. */
int mopar_model_cut_tensors(mopar_model_t model, int32_t node, int32_t* tids, int32_t cap, int32_t* count);

/* ------------------------------------------------------------------------ */
/* Slice pipeline across requests                                           */
/* ------------------------------------------------------------------------ */

/* The paper deploys every slice as its own function and scales functions by
 * running more instances, so consecutive requests occupy different slices
 * and different instances at the same time (Sec. II-A, III-A, III-C).  On one
 * GPU the pipeline keeps `replicas` instances of the sliced model; instance r
 * runs slice s on streams[r * n_slices + s] (a caller may pass one stream for
 * several slices of an instance) with its own workspace.  Batch i goes to
 * instance i mod replicas and flows through its slices; slice s starts after
 * slice s-1 of the same batch has encoded its boundary, which it decodes from
 * a ring of `depth` code buffers per (instance, cut).  Every batch runs
 * exactly the kernels of mopar_model_forward, so its output is bitwise
 * identical to the sequential forward.
 *
 * streams:   replicas * n_slices caller-owned hipStream_t (default priority).
 * ws:        mopar_pipeline_workspace_bytes(replicas) bytes, used by no one
 *            else while the pipeline lives.
 * code_bufs: replicas * depth * B device buffers, B = the plan's boundary
 *            tensors (as for mopar_model_forward); the buffer of (instance r,
 *            ring slot q, boundary tensor b) is at [(r * depth + q) * B + b],
 *            each of mopar_boundary_code_bytes of its tensor.
 * codecs:    B codecs (copied).  The plan is copied.
 * Per-op timing is not recorded by pipelined batches.
 * Errors: as mopar_model_forward; MOPAR_E_HIP if an event cannot be made. */
typedef struct mopar_pipeline_s* mopar_pipeline_t;

int mopar_pipeline_workspace_bytes(mopar_model_t model, const mopar_plan* plan, int32_t replicas, size_t* bytes);
int mopar_pipeline_create(mopar_model_t model, const mopar_plan* plan, const mopar_codec* codecs, int32_t replicas,
                          int32_t depth, void* const* streams, void* ws, size_t ws_bytes, void* const* code_bufs,
                          mopar_pipeline_t* out);

/* Enqueue one batch: read `in_dev` (the model input), write `out_dev`.  The
 * batch runs on the pipeline's own streams and does not wait for any other
 * stream: `in_dev` must already hold the input when the first slice's stream
 * reaches this batch (e.g. make that stream wait for an event recorded after
 * the input was written).  Both buffers must stay untouched by the caller
 * until the last slice's stream has finished this batch (e.g. synchronise
 * that stream).  Never blocks. */
int mopar_pipeline_submit(mopar_pipeline_t pipe, const void* in_dev, void* out_dev);

/* Graph replay (HIP graphs; off by default).  With `enable` set, each later
 * mopar_pipeline_submit replays an executable graph of the batch's kernels
 * instead of launching them one by one: the graph of a (ring slot, in_dev,
 * out_dev) triple is captured from the instance's stream the first time that
 * triple is submitted (nothing runs during capture) and kept until the
 * pipeline is destroyed or graphs are disabled; each distinct triple adds one
 * graph.  Replays run exactly the kernels of an ordinary submit, so outputs
 * are bitwise identical.  Needs every instance to run all of its slices on one
 * stream (the cross-stream events are then implied by stream order):
 * otherwise MOPAR_E_UNSUPPORTED.  `enable` = 0 destroys the cached graphs --
 * only once the batches submitted with them have finished.
 * Errors: MOPAR_E_ARG (null pipeline), MOPAR_E_UNSUPPORTED, and MOPAR_E_HIP
 * from a later submit if capture or instantiation fails. */
int mopar_pipeline_use_graphs(mopar_pipeline_t pipe, int32_t enable);

/* Destroy the pipeline's events; the caller must have synchronised its streams. */
void mopar_pipeline_destroy(mopar_pipeline_t pipe);

/* ------------------------------------------------------------------------ */
/* Measurement                                                               */
/* ------------------------------------------------------------------------ */

/* Per-op timing.  While enabled, every kernel that an op of
 * mopar_slice_forward / mopar_model_forward launches (an LSTM op counts as
 * one op, all its launches included), and every kernel of a boundary encode /
 * decode of mopar_model_forward, is launched with its own pair of HIP events
 * that the runtime stamps with that kernel's start and end on the device.  A
 * slot's time is the sum of its kernels' durations: launch gaps between
 * kernels are not counted.  Events are created on first use and reused (no
 * device memory); disabling destroys them.  Not thread-safe with respect to
 * concurrent forwards on the same model. */
int mopar_model_set_timing(mopar_model_t model, int32_t enable);

/* Number of timing slots: n_ops + 2 * (n_layers - 1).  Slot i < n_ops is op
 * i; slot n_ops + 2*c is the encode and n_ops + 2*c + 1 the decode of cut c
 * (the c-th split point of the last forward). */
int mopar_model_timing_slots(mopar_model_t model, int32_t* n);

/* Wait for the events of the last timed forward and write each slot's
 * duration in milliseconds to ms[0..n-1] (-1 for slots that did not run). */
int mopar_model_op_times(mopar_model_t model, float* ms, int32_t n);

/* Measured layer profile for the parallelism search of Alg. 1 (the t_p(l, eta)
 * of Eq. 5, Sec. III-C).  For eta = 1 .. k_max the whole model runs as one
 * slice with min(eta, RD width) sub-slices on every node that has an RD op
 * (1 elsewhere): one warm-up pass, then `reps` timed passes with per-kernel
 * device timing (as mopar_model_set_timing).  tp_out[l * k_max + eta - 1]
 * receives the median over the passes of node l's summed kernel time, in
 * seconds.  Sub-slices write their own output columns of the shared tensor,
 * so the matching aggregation table t_a is zero.  Feed tp_out (and
 * tp_out[l * k_max] as each node's time_s) to mopar_plan_slices.
 *   in_dev / out_dev: model input and output (device; out is overwritten);
 *   ws: workspace of at least mopar_model_workspace_bytes bytes;
 *   k_max 1..64, reps 1..1000.
 * Runs on `stream` and returns once its events have completed (synchronous
 * for the host).  Per-op timing is left as it was before the call. */
int mopar_model_measure(mopar_model_t model, int32_t k_max, int32_t reps, const void* in_dev, void* out_dev,
                        void* ws, size_t ws_bytes, void* stream, double* tp_out);

/* Description of the last error on this thread ("" when none). */
const char* mopar_last_error(void);

/* Library version string. */
const char* mopar_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MOPAR_H */
