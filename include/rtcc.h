/*
 * rtcc.h - C ABI of the release-triggered fork-join detector library.
 *
 * The library runs the edge-side DNN of release-triggered communication-
 * computation coupling (RTCC) on one AMD Instinct MI355X (gfx950):
 *
 *   per agent k (branch encoder E_k, independent of the other agents):
 *     pinned host staging -> H2D copy -> pillar cell ids -> counting sort by
 *     cell -> point-feature net + dense canvas -> 3x3 conv backbone ->
 *     upsample + concat into agent slot k
 *   join (all K encoders finished):
 *     pose warp to the ego frame -> cross-agent fusion (max or attention)
 *     -> 1x1 detection head -> threshold + box decode -> D2H
 *
 * Paper: "Uplink-Completion-Triggered Edge-GPU Inference for Multi-Agent
 * Cooperative Perception" (arXiv 2608.08330).
 *   - completion event e_k = Complete(k, a_k)           Sec. IV-B, eq. completion_event
 *   - branch state machine WAITING->RELEASED->RUNNING->FINISHED
 *                                                       Sec. IV-C, eq. branch_state
 *   - validation, ready order (r_k, k), rejection of duplicate, premature,
 *     malformed or inconsistent events                  Sec. IV-C
 *   - release certificate r_k = a_k, release causality  eqs. release_certificate,
 *                                                       release_causality
 *   - communication-infeasible frame: fusion withheld   Sec. IV-C, Alg. 1
 *   - fixed agent-indexed feature slots, post-join subgraph after all K
 *     encoders are FINISHED                             Sec. IV-D
 *   - pinned staging, async H2D, event-gated encoder    Sec. IV-F
 *   - Barrier baseline: all encoders released at A = max_k a_k   Sec. V
 *   - node service times by event timing after warm-up  Sec. IV-A, Sec. V-A1
 *
 * Conventions for every call:
 *   - Every function returns rtcc_status (RTCC_OK == 0) except
 *     rtcc_destroy, rtcc_status_str and rtcc_last_error.  No C++ exception
 *     crosses the ABI.  On error, rtcc_last_error(ctx) describes the cause.
 *   - Pointers named host_* point to host memory, device_* to device memory
 *     of the context's HIP device.  The library never frees memory it did
 *     not allocate; pointers it returns stay owned by the context.
 *   - Times are seconds, as double.  t0 and "now" are CLOCK_MONOTONIC.
 *   - One context drives one GPU.  Calls on one context are serialised by an
 *     internal mutex; release calls for different agents may come from
 *     different threads.
 */
#ifndef RTCC_H
#define RTCC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Only the functions below are exported; the library is built with hidden
 * default visibility. */
#if defined(__GNUC__) || defined(__clang__)
#define RTCC_API __attribute__((visibility("default")))
#else
#define RTCC_API
#endif

#define RTCC_ABI_VERSION 6
#define RTCC_MAX_AGENTS 16
#define RTCC_MAX_STAGES 4

typedef enum rtcc_status {
    RTCC_OK = 0,
    RTCC_E_ARG = 1,        /* bad argument, inconsistent descriptor, size mismatch */
    RTCC_E_STATE = 2,      /* call not valid in the current frame state           */
    RTCC_E_DUPLICATE = 3,  /* second completion event for one agent in a frame    */
    RTCC_E_MALFORMED = 4,  /* payload or event fails validation                   */
    RTCC_E_PREMATURE = 5,  /* event claims an arrival time later than now         */
    RTCC_E_INFEASIBLE = 6, /* join while a branch is undelivered: no fusion runs  */
    RTCC_E_NOMEM = 7,      /* host or device allocation failed                    */
    RTCC_E_HIP = 8,        /* HIP runtime error (message in rtcc_last_error)      */
    RTCC_E_INTERNAL = 9
} rtcc_status;

typedef enum rtcc_precision { RTCC_PREC_FP32 = 0, RTCC_PREC_BF16 = 1 } rtcc_precision;
typedef enum rtcc_fusion { RTCC_FUSE_MAX = 0, RTCC_FUSE_ATTN = 1 } rtcc_fusion;

/* Release rule.  RELEASE (RTCC): r_k = a_k, each branch is dispatched by its
 * own completion event.  BARRIER: events are validated and recorded (the
 * branch stays WAITING); the K-th valid event releases all K encoders at A,
 * dispatched together in (A, k) = index order. */
typedef enum rtcc_mode { RTCC_MODE_RELEASE = 0, RTCC_MODE_BARRIER = 1 } rtcc_mode;

/* Executor.  PER_BRANCH_STREAMS: one HIP stream per agent plus a join
 * stream.  SERIAL: one compute stream for every encoder and the post-join
 * subgraph (the single-stream model of Sec. III-B), plus a copy stream. */
typedef enum rtcc_exec { RTCC_EXEC_PER_BRANCH_STREAMS = 0, RTCC_EXEC_SERIAL = 1 } rtcc_exec;

/* Branch state z_k (Sec. IV-C eq. branch_state, Alg. 1).  WAITING: input
 * not complete, or (BARRIER) recorded but not yet released; RELEASED: input
 * validated and encoder enqueued on the device; RUNNING: the device has
 * reached the encoder (its input copy and earlier work of its stream are
 * done); FINISHED: the encoder completed and its slot is stored. */
typedef enum rtcc_branch_state {
    RTCC_WAITING = 0,
    RTCC_RELEASED = 1,
    RTCC_RUNNING = 2,
    RTCC_FINISHED = 3
} rtcc_branch_state;

typedef struct rtcc_stage {
    int32_t stride;  /* stride of the stage's first 3x3 conv (1 or 2) */
    int32_t c_out;   /* output channels of every conv of the stage    */
    int32_t n_convs; /* number of 3x3 convs in the stage (>= 1)       */
} rtcc_stage;

/* Network and geometry.  Grid: W = round((x_max - x_min) / pillar_size),
 * H likewise from y.  A point is kept iff x, y, z, r are finite,
 * x_min <= x < x_max (same for y, z) and its float32 index
 * floor((x - x_min) / pillar_size) lies in [0, W) (same for y).
 * Channel counts must be multiples of 32; c_pfn <= 64 * 8. */
typedef struct rtcc_model_desc {
    int32_t abi_version;           /* RTCC_ABI_VERSION                          */
    int32_t n_agents;              /* K, 1..RTCC_MAX_AGENTS; agent 0 is the ego */
    int64_t max_points;            /* N_max points per agent and frame          */
    float x_min, x_max, y_min, y_max, z_min, z_max; /* metres                   */
    float pillar_size;             /* metres                                    */
    int32_t max_points_per_pillar; /* points of a pillar fed to the PFN (32)    */
    int32_t c_pfn;                 /* point-feature channels                    */
    int32_t precision;             /* rtcc_precision                            */
    int32_t n_stages;              /* 1..RTCC_MAX_STAGES                        */
    rtcc_stage stages[RTCC_MAX_STAGES];
    int32_t up_channels;           /* 0: no upsampling (slot = last stage)      */
    int32_t fusion;                /* rtcc_fusion                               */
    int32_t n_anchors;             /* must be 2                                 */
    float anchor_w, anchor_l, anchor_h, anchor_z;
    float anchor_yaw[2];
    float score_logit_threshold;   /* keep anchor iff class logit > threshold   */
    /* Rotated NMS after decoding (part of T^det, Sec. V-A3): 0 = off; else the
     * first nms_max_candidates decoded boxes by score (descending, ties by
     * ascending anchor index), 1 .. 16384, take part.  A candidate is kept
     * iff its bird's-eye-view IoU (float64) with every box kept before it is
     * <= nms_iou_threshold (in [0, 1]).  Footprint of (x, y, z, w, l, h, yaw):
     * the rectangle centred at (x, y), side l along the heading, w across;
     * a box with a non-finite footprint or w, l <= 0 overlaps nothing. */
    int32_t nms_max_candidates;
    float nms_iou_threshold;
    /* Placement of the pose warp.  0: in the post-join subgraph, fused with
     * the cross-agent fusion.  1: as the last node of every branch, which
     * resamples its slot on the ego grid and stores the ego-frame map in the
     * activation dtype (RTCC_T_WARPED); the join then only fuses the K maps.
     * The warp of agent k needs only E_k's slot and k's pose, so both
     * placements keep the DAG's dependencies (Sec. III-B); with max fusion
     * they give identical outputs, with attention they differ by the rounding
     * of the stored maps (bf16). */
    int32_t warp_in_branch;
    /* Fusion shape.  0: each branch upsamples and concatenates its stage
     * outputs into its slot; the join fuses the K slots.  1 (multi-scale, the
     * paper's post-join subgraph of multi-scale fusion, upsampling,
     * concatenation and heads, Sec. III-B): each branch ends at its stage
     * outputs; the join warps every agent's stage-s map onto the stage-s ego
     * grid (H_s x W_s cells covering the BEV region), fuses the K maps of
     * each scale (RTCC_T_FUSED_STAGE), upsamples each fused map once into the
     * concatenated feature map (RTCC_T_FUSED) and runs the head.  Needs
     * up_channels > 0 and warp_in_branch = 0. */
    int32_t multiscale;
} rtcc_model_desc;

/* Optional device-memory hook: every device buffer of a context (weights,
 * activations, slots, scratch) comes from dev_alloc and goes back through
 * dev_free at rtcc_destroy, e.g. PyTorch's caching allocator.  dev_alloc
 * returns NULL on failure (rtcc_create then fails with RTCC_E_NOMEM); the
 * memory must stay valid until dev_free.  Pinned host staging is always
 * hipHostMalloc. */
typedef void *(*rtcc_dev_alloc_fn)(size_t bytes, void *user);
typedef void (*rtcc_dev_free_fn)(void *ptr, void *user);

typedef struct rtcc_runtime_opts {
    int32_t exec;          /* rtcc_exec                                              */
    int32_t use_graphs;    /* 1: each branch's encoder (after the input copy) and the
                              post-join subgraph (split at T^head) run as HIP graphs,
                              captured on first use and updated in place when a
                              branch's point count, input pointer or pose, or the
                              join's poses, change; not while node_timing = 1          */
    int32_t node_timing;   /* 1: record HIP events around every node of every frame  */
    int32_t device;        /* HIP device ordinal                                     */
    double premature_tol_s;/* an event with arrival_t > now - t0 + tol is premature  */
    /* Tiling override of the 3x3 convolutions (tests and tuning; results are
     * the same function of the inputs, within rounding of the summation
     * order): 0 = the per-layer plan; 1..6 = that halo tiling (1: 8 x 16
     * pixels x 128 channels, 2: 4 x 16 x 128, 3 / 4: the stride-2 forms of 1
     * / 2, 5: 4 x 16 x 64 in two wave groups, 6: its stride-2 form, 8: 1
     * with 64-byte channel chunks at any channel count, 9: 16 x 16 x 128,
     * 10: 9 with 64-byte chunks, 11: the stride-2 8 x 16 x 256) on every
     * layer whose stride and channels it supports, the plan elsewhere; 7 =
     * the implicit GEMM on every layer, 12 = the implicit GEMM with 256 x
     * 128 tiles (every other tile summing its K steps in reverse order) on
     * every layer with 128k output channels.  conv_splits (0
     * or 1: none) splits the K loop of the forced layers where it divides
     * evenly.  Values outside [0, 12]: RTCC_E_ARG. */
    int32_t conv_variant;
    int32_t conv_splits;
    rtcc_dev_alloc_fn dev_alloc;  /* NULL: hipMalloc / hipFree                     */
    rtcc_dev_free_fn dev_free;    /* required with dev_alloc                       */
    void *alloc_user;             /* passed to dev_alloc / dev_free                */
    /* Optional hipStream_t of the context's device on which the post-join
     * subgraph (and, with the SERIAL executor, every encoder) runs, e.g. the
     * caller's PyTorch stream; NULL: a stream of the context's own.  Not
     * destroyed by the library. */
    void *join_stream;
} rtcc_runtime_opts;

typedef struct rtcc_detections {
    int64_t count;            /* number of detections (after NMS when it is on)         */
    int64_t count_decoded;    /* anchors above the score threshold, before NMS          */
    const float *boxes;       /* [count][7] x, y, z, w, l, h, yaw (ego frame, m / rad)  */
    const float *scores;      /* [count] sigmoid of the class logit                     */
    const int32_t *anchor_idx;/* [count] ascending (row * W2 + col) * 2 + anchor        */
    double t_head_s;          /* raw head outputs on the GPU, seconds since t0          */
    double t_det_s;           /* detections on the host, seconds since t0               */
    int32_t n_agents;
    double arrival_s[RTCC_MAX_AGENTS];  /* a_k as given in the completion events        */
    double dispatch_s[RTCC_MAX_AGENTS]; /* host time the branch was enqueued, since t0  */
} rtcc_detections;

typedef enum rtcc_tensor_id {
    RTCC_T_PILLAR_CELLS = 0,  /* int32 [P] non-empty cells, ascending             (agent) */
    RTCC_T_PILLAR_COUNTS = 1, /* int32 [P] points per pillar (before the 32 cap)  (agent) */
    RTCC_T_CANVAS = 2,        /* [H, W, c_pfn] stored dtype                        (agent) */
    RTCC_T_SLOT = 3,          /* [H2, W2, C] stored dtype, agent slot (E_ARG when
                                 multiscale = 1: the branch ends at its stages)      (agent) */
    RTCC_T_FUSED = 4,         /* [H2, W2, C] stored dtype, the head's input                 */
    RTCC_T_HEAD = 5,          /* float32 [H2, W2, 16]                                       */
    RTCC_T_STAGE_OUT = 6,     /* [Hs, Ws, Cs] stored dtype, last conv of stage `agent>>8`,
                                 agent `agent & 255`                                        */
    RTCC_T_DECODED = 7,       /* float32 [count_decoded][9] before NMS: x, y, z, w, l, h,
                                 yaw, score, anchor index (int32 bits); ascending anchor    */
    RTCC_T_WARPED = 8,        /* [H2, W2, C] stored dtype, the agent's ego-frame map when
                                 warp_in_branch = 1 (E_ARG otherwise)               (agent) */
    RTCC_T_FUSED_STAGE = 9,   /* [Hs, Ws, Cs] stored dtype, fused map of stage `agent` when
                                 multiscale = 1 (E_ARG otherwise)                           */
    RTCC_T_PILLAR_MEMBERS = 10,/* int32 [sum_p min(count_p, max_points_per_pillar)]: the
                                 points each pillar fed to the PFN, as original indices,
                                 pillar by pillar in ascending cell order, ascending
                                 within a pillar (the order inside a pillar's segment on
                                 the device is arbitrary; this readback sorts it)   (agent) */
    RTCC_T_CONV_OUT = 11      /* [Ho, Wo, Co] stored dtype, output of 3x3 conv layer
                                 `agent >> 8` (0-based over all stages), agent
                                 `agent & 255`                                              */
} rtcc_tensor_id;

typedef struct rtcc_ctx rtcc_ctx;

/* Create a context: validate the descriptor, convert and upload the
 * weights, allocate pinned staging, device slots and activations for every
 * agent (no memory is shared between agents), create streams and events.
 *
 * weights: float32, little endian, tensors back to back in this order
 * (Sec. IV-A: the trained DNN's parameters, here a seeded network):
 *   pfn_w [4][c_pfn], pfn_b [c_pfn]
 *   for each stage s, conv l: w [3][3][C_in][C_out] (HWIO), b [C_out]
 *   if up_channels: for each stage s: w [u][u][C_s][up] with u = product of
 *     the strides of stages 1..s, b [up]
 *   head_w [C][16], head_b [16], C = up_channels * n_stages or the last
 *     stage's channels; the 16 outputs are 2 anchors x (logit, 7 residuals).
 * The buffer is borrowed for the call only; weights_bytes must equal the
 * exact size.  bf16 workloads round weight matrices to bfloat16 (RNE);
 * biases stay float32.  opts may be NULL (defaults: per-branch streams, no
 * graphs, no node timing, device 0, tolerance 1e-6 s).
 * Errors: RTCC_E_ARG, RTCC_E_NOMEM, RTCC_E_HIP. */
RTCC_API rtcc_status rtcc_create(const rtcc_model_desc *model, const void *weights, size_t weights_bytes,
                        const rtcc_runtime_opts *opts, rtcc_ctx **out);

/* Weights checkpoint: the blob of rtcc_create with a manifest that names it
 * (the paper's detector loads trained parameters, Sec. IV-A; here the
 * parameters are a seeded draw, and the manifest says which).  Little
 * endian, in this order:
 *   header, 128 bytes:
 *     [0, 8)     magic "RTCCWGT" and a NUL byte
 *     [8, 12)    uint32 version = 1
 *     [12, 16)   uint32 n_tensors, in [1, 4096]
 *     [16, 48)   config id: text, NUL-terminated, zero-padded
 *     [48, 56)   uint64 seed of the draw the weights come from (0 if none)
 *     [56, 64)   uint64 data_offset: start of the data section, a multiple
 *                of 64, after the tensor table (the gap is zero)
 *     [64, 72)   uint64 data_bytes: the data section runs to the end of the
 *                file (data_offset + data_bytes = file size)
 *     [72, 104)  SHA-256 (FIPS 180-4) of the data section
 *     [104, 128) zero
 *   tensor table, n_tensors entries of 128 bytes, in data order:
 *     [0, 64)    name, NUL-terminated, zero-padded
 *     [64, 68)   uint32 dtype = 0 (float32)
 *     [68, 72)   uint32 ndim in [1, 4]
 *     [72, 104)  int64 shape[4] (entries past ndim are 0)
 *     [104, 112) uint64 offset of the tensor in the data section
 *     [112, 120) uint64 nbytes = 4 x the product of the shape
 *     [120, 128) zero
 *   data section: the tensors back to back with no gaps, which is exactly
 *     the weights blob of rtcc_create (names and shapes as listed there:
 *     pfn_w, pfn_b, s{s}c{l}_w / _b, up{s}_w / _b, head_w, head_b). */
typedef struct rtcc_checkpoint_info {
    char config_id[32];
    uint64_t seed;
    int32_t version;
    int32_t n_tensors;
    uint64_t data_bytes;
    uint8_t sha256[32];      /* of the data section, as verified                */
} rtcc_checkpoint_info;

/* Parse and verify a checkpoint held in host memory (borrowed for the
 * call): header, table, exact size and the data section's SHA-256.
 * Errors: RTCC_E_ARG (NULL pointer), RTCC_E_MALFORMED (any check fails;
 * rtcc_last_error(NULL) names it).  On error *info is zeroed. */
RTCC_API rtcc_status rtcc_read_checkpoint(const void *file, size_t file_bytes, rtcc_checkpoint_info *info);

/* rtcc_create from a checkpoint: verified as by rtcc_read_checkpoint, and
 * its tensor table must list the descriptor's tensors in blob order with
 * their names and shapes (RTCC_E_ARG otherwise).  The file is borrowed for
 * the call only.  Other errors as rtcc_create. */
RTCC_API rtcc_status rtcc_create_from_checkpoint(const rtcc_model_desc *model, const void *file, size_t file_bytes,
                                                 const rtcc_runtime_opts *opts, rtcc_ctx **out);

/* Release everything the context owns.  NULL is a no-op. */
RTCC_API void rtcc_destroy(rtcc_ctx *ctx);

/* Select the release rule for the following frames.  RTCC_E_STATE inside
 * a frame (between rtcc_begin_frame and the end of rtcc_join_and_detect). */
RTCC_API rtcc_status rtcc_set_mode(rtcc_ctx *ctx, rtcc_mode mode);

/* Pinned host buffer [capacity][4] float32 (x, y, z, r) of one agent, owned
 * by the context and valid until rtcc_destroy.  Branch inputs stay in
 * pinned host memory until their arrival (Sec. IV-F): fill it before the
 * completion event and pass it to rtcc_release_branch to avoid a host copy. */
RTCC_API rtcc_status rtcc_staging_buffer(rtcc_ctx *ctx, int32_t agent, float **pinned, int64_t *capacity);

/* Start a frame: every branch WAITING, outputs cleared, t0 = uplink start. */
RTCC_API rtcc_status rtcc_begin_frame(rtcc_ctx *ctx, double t0_monotonic_s);

/* Completion event e_k = Complete(agent, arrival_t) (Sec. IV-B/IV-C).
 *   host_points: [n][4] float32 in the agent's own frame; if it is the
 *     agent's staging buffer nothing is copied, otherwise it is copied into
 *     staging before the call returns (the caller keeps ownership).
 *   pose: agent-to-ego SE(2) (yaw rad, tx m, ty m): p_ego = R(yaw) p + t.
 *   arrival_t: a_k in seconds since t0.
 * Checks, in order: E_STATE (no open frame), E_ARG (agent not in [0, K)),
 * E_DUPLICATE (branch not WAITING), E_MALFORMED (n < 0, n > max_points,
 * NULL points with n > 0, non-finite pose or arrival, arrival < 0),
 * E_PREMATURE (now - t0 < arrival_t - tol).  A rejected event leaves the
 * branch WAITING.  RELEASE mode: enqueue the H2D copy and encoder E_k on
 * the branch stream and return without waiting.  BARRIER mode: record;
 * the K-th valid event enqueues all branches, as one group (see
 * rtcc_release_branches).  If an enqueue fails (E_HIP / E_NOMEM), the
 * branches of that enqueue stay WAITING and the frame's join returns
 * E_STATE. */
RTCC_API rtcc_status rtcc_release_branch(rtcc_ctx *ctx, int32_t agent, const float *host_points, int64_t n,
                                const float pose[3], double arrival_t);

/* Same event for an input that is already resident in device memory (the
 * resident-input runs of Sec. V-B).  device_points [n][4] float32 must stay
 * valid and unmodified until rtcc_join_and_detect returns, and any writes
 * to it must be complete (e.g. the producing stream synchronised) before
 * the call. */
RTCC_API rtcc_status rtcc_release_branch_device(rtcc_ctx *ctx, int32_t agent, const float *device_points,
                                       int64_t n, const float pose[3], double arrival_t);

/* One completion event of a batch (rtcc_release_branches). */
typedef struct rtcc_event {
    int32_t agent;
    int32_t device;        /* 0: points in host memory (as rtcc_release_branch),
                              1: resident in device memory (as
                              rtcc_release_branch_device)                       */
    const float *points;   /* [n][4] float32, agent frame                       */
    int64_t n;
    float pose[3];         /* agent-to-ego SE(2): yaw rad, tx m, ty m           */
    double arrival_t;      /* a_k, seconds since t0                             */
} rtcc_event;

/* Completion events that arrived together (Sec. IV-B/IV-C: every e_k that
 * has arrived releases its branch; several may arrive at once).  The events
 * are checked and recorded in array order exactly as count calls of
 * rtcc_release_branch / rtcc_release_branch_device would be (a second event
 * for one agent within the batch is E_DUPLICATE); status, if not NULL,
 * receives each event's result [count].  RELEASE mode: the branches of all
 * accepted events are released as one group: their encoders' pillar stage
 * runs as one launch chain over the group (one grid row per agent) and each
 * backbone then continues on its own branch stream; the outputs are those
 * of separate releases, bit for bit.  BARRIER mode: the events are
 * recorded, and when the K-th valid event is among them all K branches are
 * released as one group.  Returns RTCC_OK if every event was accepted and
 * enqueued; otherwise an enqueue failure (E_HIP / E_NOMEM: the whole group
 * stays WAITING and the frame's join returns E_STATE), else the first
 * rejected event's status; rtcc_last_error names it.  E_ARG if count is not
 * in [0, RTCC_MAX_AGENTS] or events is NULL with count > 0 (nothing
 * recorded). */
RTCC_API rtcc_status rtcc_release_branches(rtcc_ctx *ctx, int32_t count, const rtcc_event *events,
                                           rtcc_status *status);

/* Join and detect.  If any branch's input is undelivered the frame is
 * communication-infeasible: RTCC_E_INFEASIBLE, no fusion kernel is
 * launched and the frame is closed.  If every input arrived but an
 * encoder's enqueue failed: RTCC_E_STATE, likewise without fusion.
 * Otherwise wait (on the GPU) for every
 * encoder, run warp, fusion, head, decode and (if enabled) rotated NMS, copy
 * the detections to the host and block until they are there.  out's arrays belong to the
 * context and stay valid until the next rtcc_begin_frame. */
RTCC_API rtcc_status rtcc_join_and_detect(rtcc_ctx *ctx, rtcc_detections *out);

/* State of one branch in the current or last frame (rtcc_branch_state);
 * RUNNING and FINISHED are read from the device without blocking. */
RTCC_API rtcc_status rtcc_get_branch_state(rtcc_ctx *ctx, int32_t agent, int32_t *state);

/* Size in bytes of a tensor of the last completed frame (see
 * rtcc_tensor_id for which take an agent). */
RTCC_API rtcc_status rtcc_tensor_bytes(rtcc_ctx *ctx, int32_t id, int32_t agent, size_t *bytes);

/* Copy a tensor of the last completed frame to host memory dst of exactly
 * rtcc_tensor_bytes bytes (E_ARG otherwise).  Blocks until copied. */
RTCC_API rtcc_status rtcc_get_tensor(rtcc_ctx *ctx, int32_t id, int32_t agent, void *dst, size_t bytes);

/* Node service times c_v (Sec. IV-A): re-run the last completed frame's
 * work node by node on one stream, `warmup` untimed passes then `reps`
 * timed passes, and write the median of each node in ms.  Nodes: E_0 ..
 * E_{K-1} (encoder without the H2D copy, with the warp when
 * warp_in_branch = 1), then the post-join subgraph (warp + fusion, or
 * fusion alone, + head + decode + rotated NMS when it is on).  *n_nodes is
 * K + 1; median_ms must hold RTCC_MAX_AGENTS + 1 floats. */
RTCC_API rtcc_status rtcc_profile_nodes(rtcc_ctx *ctx, int32_t warmup, int32_t reps, float *median_ms,
                               int32_t *n_nodes);

/* Per-kernel-group GPU durations (ms) of the last frame, recorded when
 * opts.node_timing = 1.  For each agent k, in order: h2d, pillar (cell ids,
 * counting sort, segment), pfn_canvas, conv[0 .. L-1], up[0 .. S-1] (0 if
 * no upsampling; 0 each when multiscale = 1), warp (0 unless warp_in_branch
 * = 1 and the agent's pose is not the identity, which needs no
 * resampling); then warp_fuse (or fuse; with multiscale = 1 the warp and
 * fusion of every scale and the upsampling of the fused maps), head,
 * decode, nms (0 if off).  Conv nodes, the branch warp and a one-kernel
 * warp_fuse / fuse node are the execution time of their kernels (events
 * that bracket the kernels themselves); the other nodes span the stream
 * between events recorded around them, dispatch gaps included.  *n = number written; ms must hold
 * at least rtcc_node_count() floats. */
RTCC_API rtcc_status rtcc_node_times(rtcc_ctx *ctx, float *ms, int32_t *n);
RTCC_API rtcc_status rtcc_node_count(rtcc_ctx *ctx, int32_t *n);

/* Kernel tiling of 3x3 conv layer `layer` (0-based over all stages):
 * plan[0] = 0 implicit GEMM, 12 its 256 x 128 tiles, 1..6 and 8..11 the
 * halo tilings of rtcc_runtime_opts.conv_variant for a launch over one
 * agent's map (a batched launch over several agents may use a wider tiling
 * of the same accumulation order: 1 or 9 for 2, 3 or 11 for 3 and 4, 10
 * for 8); plan[1] = K slices (1 = unsplit).  plan:
 * caller-owned int32_t[2].  Errors: RTCC_E_ARG (NULL or layer out of
 * range), RTCC_E_STATE (the host test library has no kernels). */
RTCC_API rtcc_status rtcc_conv_plan(rtcc_ctx *ctx, int32_t layer, int32_t *plan);

/* The tiling the library plans for a 3x3 conv layer, without a context or a
 * device: shape = {Hi, Wi, C_in, Ho, Wo, C_out, stride, n_cu} (int32_t[8],
 * n_cu = the GPU's compute units; a context plans with its device's count),
 * bf16 != 0 for bf16 operands (else fp32), maps = the agents' maps one
 * launch covers (1: one agent; a group release launches every layer over
 * its members).  out[0] = tiling id as in rtcc_conv_plan (a launch over
 * several maps may take a wider tiling of the same accumulation order),
 * out[1] = K slices.  out: caller-owned int32_t[2].  Errors: RTCC_E_ARG
 * (NULL pointer, a size or n_cu below 1, stride not 1 or 2, maps outside
 * [1, 16]). */
RTCC_API rtcc_status rtcc_conv_tiling(int32_t bf16, const int32_t *shape, int32_t maps, int32_t *out);

/* With opts.use_graphs = 1: counts[0] = HIP graphs instantiated, counts[1] =
 * in-place updates attempted (a branch or the join whose arguments changed
 * since its graph was captured is captured again and the executable graph
 * updated; a failed update instantiates anew), counts[2] = graph launches,
 * all since rtcc_create (zeros without graphs).  counts: caller-owned
 * int64_t[3].  Errors: RTCC_E_ARG (NULL ctx or counts). */
RTCC_API rtcc_status rtcc_graph_stats(rtcc_ctx *ctx, int64_t *counts);

/* Rotated NMS of caller-provided decoded boxes, the same kernels that end
 * rtcc_join_and_detect (Sec. V-A3: decoding, score thresholding and rotated
 * NMS end T^det).  On the current HIP device, synchronous.
 *   device_records: [n][9] float32 x, y, z, w, l, h, yaw, score, anchor
 *     index (int32 bit pattern), in ascending anchor index (ties in score
 *     rank by it); any non-NaN score ranks by its value (negative scores,
 *     raw logits for instance, included; -0 equals +0).  Every write to the
 *     records must be complete before the call (synchronise the stream that
 *     produced them): the call runs on a stream of its own;
 *   max_candidates, iou_threshold: as nms_max_candidates / nms_iou_threshold
 *     of rtcc_model_desc (1 .. 16384, [0, 1]);
 *   device_out: [min(n, max_candidates)][9] float32, receives the kept
 *     records in ascending anchor index; *kept their number.
 * n = 0 keeps nothing.  E_ARG for NULL pointers with n > 0, n < 0,
 * n > 2^31 - 1, parameters out of range, or a NaN score (found on the
 * device; device_out is then undefined); E_NOMEM / E_HIP for device
 * errors.  Scratch memory is allocated and freed inside the call.  The
 * message of a failure is rtcc_last_error(NULL). */
RTCC_API rtcc_status rtcc_rotated_nms(const float *device_records, int64_t n, int32_t max_candidates,
                                      float iou_threshold, float *device_out, int64_t *kept);

/* rtcc_rotated_nms for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same kernels and results, with the scratch in one
 * library-owned device array of fixed size (11.9 MB per GPU, held from the
 * first call on that GPU until the process ends).  Allocates nothing and
 * creates no stream.
 *   device_records, n, max_candidates, iou_threshold, device_out, kept: as
 *     for rtcc_rotated_nms, with n <= 131072 and max_candidates <= 4096
 *     (E_ARG beyond these limits);
 *   hip_stream: a hipStream_t of the current device (NULL = the null
 *     stream); the kernels run on it, after the work already queued there,
 *     and the call returns once it has finished them.
 * Calls on one GPU share its scratch array: the library serialises them (a
 * per-device lock held until the stream is done), so a call waits for any
 * other in the process on that GPU.  The array keeps the last call's
 * contents; every part a call reads is written by that call first. */
RTCC_API rtcc_status rtcc_rotated_nms_noalloc(const float *device_records, int64_t n, int32_t max_candidates,
                                              float iou_threshold, float *device_out, int64_t *kept,
                                              void *hip_stream);

/* ------------------------------------------------------------------------
 * Host-side models of the communication and of the profiled DAG.  They run
 * on the host only (no GPU work, no context), are deterministic, and report
 * failures through rtcc_last_error(NULL).
 * ------------------------------------------------------------------------ */

/* Causal RB-allocation policies (Sec. III-A eq. pluggable_scheduler; Sec.
 * V-A2 eqs. evaluation_schedulers, evaluation_scores).  In slot t each RB
 * f goes to the eligible agent with the largest score, ties to the smallest
 * agent index:
 *   MAXRATE           s = R_{k,f}[t]
 *   MAXWEIGHT         s = Q_k[t] R_{k,f}[t]
 *   EARLIEST_RELEASE  s = -Q_k[t] / (Delta R_{k,f}[t]), -inf where R = 0
 *   WEIGHTED_RATE     s = w_k R_{k,f}[t]: DAGRank with w = the normalised
 *                     upward rank omega, Task-Weighted MaxRate with w = q
 *   ROUND_ROBIN       the first eligible agent after the last one served,
 *                     cycling in index order (the first RB of slot 1 from
 *                     agent 0)
 *   PROPORTIONAL_FAIR s = R_{k,f}[t] / Rbar_k, Rbar_k <- (1 - 1/W) Rbar_k +
 *                     (1/W) (rate served to k in the slot) after every slot
 * Q_k[t] is the slot-start backlog for every RB of the slot. */
typedef enum rtcc_sched {
    RTCC_SCHED_MAXRATE = 0,
    RTCC_SCHED_MAXWEIGHT = 1,
    RTCC_SCHED_EARLIEST_RELEASE = 2,
    RTCC_SCHED_WEIGHTED_RATE = 3,
    RTCC_SCHED_ROUND_ROBIN = 4,
    RTCC_SCHED_PROPORTIONAL_FAIR = 5
} rtcc_sched;

typedef struct rtcc_uplink_desc {
    int32_t slots;              /* T: slots emulated (the horizon T_max), >= 1          */
    int32_t agents;             /* K, >= 1                                               */
    int32_t rbs;                /* F, >= 1                                               */
    int32_t policy;             /* rtcc_sched                                            */
    double slot_s;              /* Delta, seconds, > 0                                   */
    const double *agent_weight; /* [K] w_k for WEIGHTED_RATE (finite); else unused       */
    double pf_window;           /* PROPORTIONAL_FAIR: W in slots, >= 1                   */
    double pf_init_rate;        /* PROPORTIONAL_FAIR: Rbar_k before slot 1, bit/s, > 0   */
} rtcc_uplink_desc;

/* Slot-level uplink emulation (Sec. III-A eqs. rb_orthogonality,
 * local_ready_constraint, slot_payload, queue_evolution, branch_arrival;
 * Sec. IV-B eq. eligible_set, completion_event).  Q_k[1] = B_k; in slot t
 * the agents with Q_k[t] > 0 and t >= l_k are eligible and every RB goes to
 * one of them by the policy; d_k[t] = Delta * (sum of the rates of the RBs
 * k holds, in ascending RB order); Q_k[t+1] = max(0, Q_k[t] - d_k[t]).
 *   rates:           host [T][K][F] bit/s, finite and >= 0
 *   payload_bits:    host [K] B_k, finite and > 0
 *   avail_slot:      host [K] l_k >= 1, or NULL for l_k = 1
 *   completion_slot: host [K] out: the slot in which Q_k reaches zero
 *                    (a_k = slot * Delta), 0 if still undelivered after T
 *                    slots (a_k = +inf: the frame is infeasible)
 *   rb_agent:        host [T][F] out or NULL: agent given each RB, -1 idle
 * Returns RTCC_E_ARG for invalid arguments (nothing written). */
RTCC_API rtcc_status rtcc_uplink_emulate(const rtcc_uplink_desc *desc, const double *rates,
                                         const double *payload_bits, const int32_t *avail_slot,
                                         int32_t *completion_slot, int32_t *rb_agent);

/* Single-stream latency of the profiled DAG for one arrival vector (Sec.
 * III-B eq. encoder_release, dag_precedence; Sec. III-C eq. full_latency;
 * Sec. IV-C eqs. rtcc_encoder_start, rtcc_encoder_finish,
 * rtcc_gpu_availability): encoders run one at a time in (r_k, k) order,
 * each from max(r_k, stream free) for encoder_ns[k]; the post-join subgraph
 * then takes post_ns.  mode RELEASE: r_k = a_k; BARRIER: r_k = A = max a_k.
 * Integer nanoseconds, so every result is exact.
 *   arrival_ns, encoder_ns: host [agents], in [0, 2^60); post_ns likewise
 *   latency_ns:     out: finish of the post-join subgraph (T)
 *   pre_arrival_ns: out or NULL: encoder time spent before A, the sum over
 *                   k of |[s_k, f_k) intersected with [0, A)| (W_pre under
 *                   RELEASE; 0 under BARRIER)
 *   start_ns:       out [agents] or NULL: encoder start times s_k
 * Returns RTCC_E_ARG for invalid arguments. */
RTCC_API rtcc_status rtcc_schedule_model(int32_t agents, const int64_t *arrival_ns, const int64_t *encoder_ns,
                                         int64_t post_ns, int32_t mode, int64_t *latency_ns,
                                         int64_t *pre_arrival_ns, int64_t *start_ns);

/* Upward rank of every node of a DAG (the DAGRank priority of Sec. V-A2):
 * rank(v) = cost(v) + max over successors w of rank(w), 0 without
 * successors, i.e. the longest path from v to an exit node, v included.
 *   cost_ns:   host [nodes], in [0, 2^60), summing to less than 2^60
 *   edge_list: host [edges][2] (u, v): v depends on u; NULL if edges == 0
 *   rank_ns:   host [nodes] out
 * Returns RTCC_E_ARG for invalid arguments, an endpoint out of range, a
 * self loop or a cycle. */
RTCC_API rtcc_status rtcc_upward_rank(int32_t nodes, const int64_t *cost_ns, int32_t edges,
                                      const int32_t *edge_list, int64_t *rank_ns);

/* Name of a status code. */
RTCC_API const char *rtcc_status_str(rtcc_status s);

/* Message of the last failed call on ctx; with ctx == NULL, the message of
 * the last failed context-free call (rtcc_create, rtcc_rotated_nms,
 * rtcc_uplink_emulate, rtcc_schedule_model, rtcc_upward_rank) on the
 * calling thread. */
RTCC_API const char *rtcc_last_error(const rtcc_ctx *ctx);

#ifdef __cplusplus
}
#endif

#endif /* RTCC_H */
