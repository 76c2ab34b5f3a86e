/*
 * ctc.h -- C ABI of the carry-through checksum inference library (gfx950).
 *
 * Carry-through checksum (Nazarevych et al., "Carry-Through Checksum: A
 * Lightweight Fault-Detection for CNN Inference at the Edge", IEEE ATS'26):
 * every convolution gives up its least important output filter to a
 * carry-through filter whose output channel is the channel-wise sum of the
 * layer's input feature maps (Sec. II-A, Fig. 1); normal filters ignore the
 * incoming checksum channel, so the checksum accumulates layer to layer; the
 * final FC layer gets one accumulated-checksum neuron that sums all of its
 * inputs (Sec. II-B); an inference whose accumulated checksum deviates from a
 * reference by more than a threshold tau is flagged and re-executed once
 * (Sec. II-B); tau comes from the fault-free distribution of the neuron
 * (Sec. II-C).
 *
 * Conventions for every entry point:
 *  - Device pointers are allocated by the caller (the library never
 *    allocates device memory); host pointers are plain host memory.
 *  - "stream" is a hipStream_t passed as void* (NULL = the null stream).
 *    Device calls only enqueue work and return; their results are visible
 *    after the stream is synchronised.
 *  - Arguments are validated before anything is enqueued; on an error
 *    nothing is launched, a non-zero ctc_status is returned and
 *    ctc_last_error() describes it.  No call aborts or throws.
 *  - Activations on the device are NHWC (channel fastest).  Weights are
 *    passed in canonical PyTorch layout, fp32, and packed by the library.
 */
#ifndef CTC_H
#define CTC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CTC_ABI_VERSION 3

typedef enum {
    CTC_OK = 0,
    CTC_ERR_ARG = -1,         /* bad pointer, size or shape */
    CTC_ERR_UNSUPPORTED = -2, /* valid request this library does not handle */
    CTC_ERR_DEVICE = -3,      /* a HIP call or kernel launch failed */
    CTC_ERR_WORKSPACE = -4,   /* workspace missing or too small */
    CTC_ERR_STATE = -5        /* call out of order (e.g. forward before bind) */
} ctc_status;

typedef enum { CTC_F32 = 0, CTC_F16 = 1 } ctc_dtype;

/* Role of a conv layer's last output channel (Sec. II-A):
 *  SUM   carry-through filter: 1 at the kernel centre on every input channel;
 *  ZERO  first conv of a residual block: the last filter is all zero, so the
 *        checksum entering the block is not counted twice (the residual add
 *        brings it back);
 *  PASS  depthwise conv or 1x1 projection shortcut: the last filter is 1 at
 *        the centre of the incoming checksum channel only (a depthwise filter
 *        cannot sum across channels; the shortcut delivers the checksum to
 *        the add);
 *  NONE  unprotected layer: parameters are left as given. */
typedef enum {
    CTC_ROLE_NONE = 0, CTC_ROLE_SUM = 1, CTC_ROLE_ZERO = 2, CTC_ROLE_PASS = 3
} ctc_role;

typedef struct {
    int32_t c_in, c_out;  /* channels */
    int32_t kh, kw;       /* kernel size, both odd */
    int32_t stride, pad;
    int32_t groups;       /* 1, or c_in == c_out == groups (depthwise) */
    int32_t in_has_ck;    /* 1: input channel c_in-1 is an incoming checksum */
    int32_t role;         /* ctc_role */
} ctc_layer_desc;

/* ---- carry-through construction (host, synchronous) -------------------- */

/* Sec. II-A and Eq. (1): applies the carry-through construction in place to
 * one conv layer's canonical fp32 parameters.
 *   w     [c_out][c_in/groups][kh][kw]
 *   bias  [c_out] or NULL
 *   bn_*  [c_out] each, or all four NULL (no batch normalisation)
 * Output-channel level: filter c_out-1 becomes the role's filter (see
 * ctc_role), its bias 0 and its BN entries the identity (mean 0, var 1,
 * gamma 1, beta 0).  Input-channel level (in_has_ck, groups == 1): the slice
 * of every other filter over input channel c_in-1 is set to 0.
 * Errors: CTC_ERR_ARG (NULL w, bad sizes), CTC_ERR_UNSUPPORTED (even kernel,
 * grouped but not depthwise). */
ctc_status ctc_build_filters(const ctc_layer_desc *desc, float *w,
                             float *bias, float *bn_mean, float *bn_var,
                             float *bn_gamma, float *bn_beta);

/* Sec. II-A (FC paragraph) and Sec. II-B: builds a protected FC layer.
 *   w_in  [out_f][in_f], b_in [out_f] or NULL (canonical fp32)
 *   input features ck_first .. ck_first+ck_count-1 hold checksum values
 *   (ck_count may be 0)
 * is_final = 0 (hidden layer): w_out/b_out are [out_f][in_f]/[out_f]; neuron
 *   out_f-1 becomes the all-ones carry-through neuron with bias 0, the other
 *   neurons get weight 0 on the checksum features.
 * is_final = 1 (classifier): w_out/b_out are [out_f+1][in_f]/[out_f+1]; the
 *   logits keep their weights except 0 on the checksum features and the
 *   extra neuron out_f is the accumulated-checksum neuron (weights 1, bias
 *   0).  b_out may be NULL only when b_in is NULL.
 * w_out may not alias w_in.  Errors: CTC_ERR_ARG. */
ctc_status ctc_build_fc(int32_t in_f, int32_t out_f, int32_t ck_first,
                        int32_t ck_count, int32_t is_final, const float *w_in,
                        const float *b_in, float *w_out, float *b_out);

/* Sec. II-C, distribution-based threshold: from n fault-free samples of the
 * accumulated-checksum neuron, ref = their mean (fp64) and tau = the k-th
 * smallest |S_i - ref| with k = n - ceil(alpha*n) + 1, so that fewer than
 * alpha*n of the samples deviate by more than tau.  Host, synchronous.
 * Errors: CTC_ERR_ARG (n < 1, alpha outside [0, 1], NULL pointer). */
ctc_status ctc_threshold_from_samples(const double *S, int64_t n,
                                      double alpha, double *ref, double *tau);

/* Sec. II-C, FI-based threshold (and the same order statistic for any
 * sample set at a given reference): tau = the k-th smallest |S_i - ref|,
 * k = n - ceil(alpha*n) + 1, with NaN deviations ordered last (as +Inf).
 * For the FI-based method S holds the accumulated-checksum values of the
 * non-critical faulty inferences of a campaign on training inputs and ref
 * the fault-free reference, so that fewer than alpha*n of them would be
 * flagged (false positives).  Host, synchronous.
 * Errors: CTC_ERR_ARG (n < 1, alpha outside [0, 1], NULL pointer). */
ctc_status ctc_threshold_at_ref(const double *S, int64_t n, double ref,
                                double alpha, double *tau);

/* ---- single layers and the detector (device, asynchronous) ------------- */

/* Sec. II-A (the carry-through filter is one more filter of an ordinary
 * convolution, so a protected layer is a plain conv whose last output
 * channel carries the checksum) and Eq. (1) (batch normalisation, folded
 * here into a per-channel scale and shift).  One convolution of the
 * protected network with its fused epilogue:
 *   y = act(scale[k] * conv(x, w)[k] + shift[k] (+ residual))
 * where scale/shift carry bias and batch normalisation folded per channel
 * (scale = gamma/sqrt(var+eps), shift = beta - mean*scale + bias*scale),
 * optionally followed, in the same kernel, by a 2x2 stride-2 max pool of
 * the stored (rounded) values.  The carry-through channel is ordinary
 * output channel c_out-1: it is computed by the same kernel in the same
 * tile as the normal channels, and pooled like any other channel.
 *   x_nhwc    [n][h][w][c_in] in dtype, c_in a multiple of 4
 *   w_packed  groups == 1: [c_out][kh][kw][c_in] in dtype (KRSC);
 *             depthwise:   [kh][kw][c_out] in dtype
 *   scale, shift [c_out] fp32
 *   residual  [n][p][q][c_out] in dtype or NULL (added before the ReLU)
 *   pool      0: y is the conv output; 2: y is its 2x2 stride-2 max pool
 *             [n][p/2][q/2][c_out] (window max of the stored values, NaN if
 *             any is NaN; only where a kernel for the shape has the pool:
 *             fp16, groups == 1, else CTC_ERR_UNSUPPORTED)
 *   y_nhwc    [n][p][q][c_out] (or pooled) in dtype, c_out a multiple of 4
 *   workspace device scratch for the fp32 partial sums of layers whose K is
 *             split over several workgroups (deep layers on small maps), or
 *             NULL; ws_bytes >= ctc_conv2d_workspace_bytes enables the
 *             split, anything smaller runs the layer unsplit.  Caller-owned;
 *             not read before this call and free again once the stream has
 *             passed it.  Overlapping calls must not share it.
 * with p = (h + 2 pad - kh)/stride + 1 and q likewise.  Zero padding
 * multiplies like any other tap.  Errors: CTC_ERR_ARG, CTC_ERR_UNSUPPORTED
 * (channel counts not multiples of 4, grouped but not depthwise, pool
 * without a pooling kernel), CTC_ERR_DEVICE. */
ctc_status ctc_conv2d_forward(const ctc_layer_desc *desc, ctc_dtype dtype,
                              int32_t n, int32_t h, int32_t w,
                              const void *x_nhwc, const void *w_packed,
                              const float *scale, const float *shift,
                              const void *residual, int32_t relu, int32_t pool,
                              void *y_nhwc, void *workspace, size_t ws_bytes,
                              void *stream);

/* Workspace bytes ctc_conv2d_forward uses for this conv (0: it never
 * splits K).  Host, synchronous.  Errors: as ctc_conv2d_forward's argument
 * checks. */
ctc_status ctc_conv2d_workspace_bytes(const ctc_layer_desc *desc,
                                      ctc_dtype dtype, int32_t n, int32_t h,
                                      int32_t w, int32_t pool, size_t *bytes);

/* Name of the kernel ctc_conv2d_forward launches for this conv (as
 * rocprofv3 lists it), copied into name[cap]; with a workspace of
 * ctc_conv2d_workspace_bytes a split layer also launches splitk_reduce.
 * Host, synchronous.  Errors: as ctc_conv2d_forward's argument checks. */
ctc_status ctc_conv2d_kernel_name(const ctc_layer_desc *desc, ctc_dtype dtype,
                                  int32_t n, int32_t h, int32_t w, int32_t pool,
                                  char *name, int32_t cap);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * convolution as ctc_conv2d_forward, same arguments, without a workspace.
 * Layers that split K keep their fp32 partial sums in a static scratch
 * array of the library (32 MiB of module memory per GPU, held from the
 * library's load until the process ends); the call allocates nothing.
 * Every call on one GPU shares that array, so calls that overlap on one
 * GPU (other streams, other host threads) race; it keeps the last call's
 * contents, none of which a later call reads.  Errors: as
 * ctc_conv2d_forward, and CTC_ERR_WORKSPACE (nothing launched) when the
 * layer's partial sums, ctc_conv2d_workspace_bytes, exceed 32 MiB. */
ctc_status ctc_conv2d_forward_noalloc(const ctc_layer_desc *desc,
                                      ctc_dtype dtype, int32_t n, int32_t h,
                                      int32_t w, const void *x_nhwc,
                                      const void *w_packed, const float *scale,
                                      const float *shift, const void *residual,
                                      int32_t relu, int32_t pool, void *y_nhwc,
                                      void *stream);

/* Sec. II-B detection for a batch: flag[i] = !(|S[i*stride] - ref| <= tau)
 * evaluated in fp32, so NaN and +-Inf are flagged.  Writes flags[batch]
 * (0/1, may be NULL), *n_flagged and idx[0 .. *n_flagged-1], the flagged
 * rows in ascending order (idx may be NULL).  All pointers are device
 * pointers; 1 <= batch <= 4096.  Errors: CTC_ERR_ARG, CTC_ERR_DEVICE. */
ctc_status ctc_verify(const float *S, int32_t batch, int32_t stride,
                      float ref, float tau, uint8_t *flags,
                      int32_t *n_flagged, int32_t *idx, void *stream);

/* ---- whole protected network ------------------------------------------ */

typedef enum {
    CTC_OP_CONV = 1, CTC_OP_MAXPOOL = 2, CTC_OP_GAP = 3, CTC_OP_FC = 4
} ctc_op_kind;

/* One layer of a network description; op i writes tensor i+1, tensor 0 is
 * the network input.  Roles are derived by the library from the structural
 * flags (Sec. II-A and its residual-network rule). */
typedef struct {
    int32_t kind;        /* ctc_op_kind */
    int32_t input;       /* tensor id read */
    int32_t residual;    /* CONV: tensor id added before the ReLU, or -1 */
    int32_t c_in, c_out; /* CONV: channels; FC: in / out features */
    int32_t k, stride, pad, groups; /* CONV; MAXPOOL uses k, stride, pad */
    int32_t has_bias, has_bn, relu;
    int32_t block_first; /* CONV: first conv of a residual block (ZERO) */
    int32_t shortcut;    /* CONV: 1x1 projection shortcut (PASS) */
    int32_t final_fc;    /* FC: the classifier (gets the extra neuron) */
    int32_t flatten_c, flatten_h, flatten_w; /* FC reading a flattened
                           CxHxW map, canonical feature order NCHW; 0s else */
    int32_t out_f32;     /* keep this op's output in fp32 in an fp16 net */
} ctc_op;

typedef struct ctc_net ctc_net;

/* Sec. II-A, output-channel level, with the paper's choice of the pruned
 * channel: in every channel group that a conv or a hidden FC produces, the
 * channel with the smallest combined L1 norm -- its filters (FC rows) where
 * the group is produced plus the 2-D input slices (FC columns; after a
 * flatten, the channel's h*w columns) that read it where the group is
 * consumed -- is swapped with the group's last channel, everywhere in the
 * group: filters, bias and BN entries of the producers, input slices of the
 * consumers.  A group is a set of tensors whose channel c is the same
 * channel: depthwise convs, pooling and residual adds tie their input and
 * output (for a residual stream every block's norms count: one channel is
 * pruned for the whole stream).  The swap is a relabelling (the
 * unprotected network computes the same function); the carry-through
 * construction of ctc_net_bind / ctc_build_filters then replaces the last
 * channel, i.e. the chosen one.  Norms are fp64 sums, each layer's slice
 * in memory order, layers added in op order; ties go to the lowest channel.
 *   ops, n_ops   the network as for ctc_net_create
 *   params       6 pointers per op (w, bias, bn mean, var, gamma, beta) to
 *                canonical fp32 arrays as for ctc_net_bind, NULL where
 *                absent; modified in place (the caller owns them)
 *   chosen       [n_ops] or NULL: the chosen channel of each op's output
 *                group, -1 where none is pruned (input group, classifier)
 * Host, synchronous.  Errors: CTC_ERR_ARG (bad op list, channel counts that
 * disagree inside a group, missing weights). */
ctc_status ctc_select_channels_l1(const ctc_op *ops, int32_t n_ops,
                                  float *const *params, int32_t *chosen);

/* Values of the `protect` argument of ctc_net_create. */
typedef enum {
    CTC_PROTECT_NONE = 0,     /* unprotected network, same kernels */
    CTC_PROTECT_REPLACE = 1,  /* Sec. II-A: the last channel of every conv
                                 and hidden FC becomes the carry-through
                                 channel (the layer keeps its width) */
    CTC_PROTECT_APPEND = 2    /* one extra carry-through channel per conv /
                                 hidden FC, widths rounded up to whole
                                 16-byte channel vectors (4 fp32, 8 fp16);
                                 nothing pruned */
} ctc_protect;

/* Sec. II-A and II-B: the protected network as a whole -- every conv and
 * hidden FC carries the checksum in its last channel (roles from the
 * structural flags: SUM, ZERO for the first conv of a residual block, PASS
 * for depthwise convs and projection shortcuts), and the classifier gets
 * the accumulated-checksum neuron whose value is checked at the end.
 * Creates a network plan (host only).  classes = outputs of the final FC
 * before protection.  protect (ctc_protect) REPLACE or APPEND applies the
 * carry-through construction at bind time and adds the
 * accumulated-checksum neuron (outputs per image: classes + 1, the last
 * being S); NONE is the unprotected network with the same kernels.  In
 * APPEND mode the library widens every conv / hidden FC (and the readers
 * of their outputs) internally; parameters, tensor ids and fault indices
 * refer to the caller's ops for ctc_net_bind and to the widened network
 * everywhere else (fault sites, tensors).  Requirements: the input has <=
 * 4 channels; every conv/FC output width except the classifier's is a
 * multiple of 4 (REPLACE, NONE); grouped convs are depthwise 3x3-type (odd
 * kernel).  Errors: CTC_ERR_ARG, CTC_ERR_UNSUPPORTED. */
ctc_status ctc_net_create(const ctc_op *ops, int32_t n_ops, int32_t in_c,
                          int32_t in_h, int32_t in_w, int32_t classes,
                          ctc_dtype dtype, int32_t protect, ctc_net **out);

/* Sec. II-B (detection, then re-execution of a flagged inference): the
 * device workspace holds what that loop needs besides the layers -- a
 * ring of staged inputs, so that a flagged image can be run again from
 * its own copy, and the detector's per-pass flag rows.
 * Device workspace needed for batches of up to max_batch images (packed
 * weights, activations of one pass, the ring of staged inputs kept for
 * re-execution, detector state).  bind also allocates a few small pinned
 * host tables (pass rows read by the kernels, detector results).
 * Errors: CTC_ERR_ARG. */
ctc_status ctc_net_workspace_bytes(const ctc_net *net, int32_t max_batch,
                                   size_t *bytes);

/* Sec. II-A, Eq. (1) and Sec. II-B: applies the carry-through
 * construction (the same as ctc_build_filters / ctc_build_fc, per op) to
 * the caller's trained parameters and deploys the result.
 * Binds parameters and workspace.  host_params holds 6 pointers per op, in
 * op order: w, bias, bn_mean, bn_var, bn_gamma, bn_beta (canonical fp32,
 * PyTorch layout; NULL where the op has none).  The library keeps its own
 * host copy (faults are applied against it), applies the construction when
 * protect is REPLACE or APPEND (APPEND first places the given parameters
 * in the widened layers: original filters at their indices, zero filters
 * and identity BN in the added channels, FC columns of the added channels
 * zero), folds BN, packs to the device layout in dtype (fp16 rounding
 * to nearest even) and copies into workspace (device, ws_bytes >= the size
 * from ctc_net_workspace_bytes, 256-byte aligned).  Synchronises `stream`.
 * Errors: CTC_ERR_ARG, CTC_ERR_WORKSPACE, CTC_ERR_DEVICE. */
ctc_status ctc_net_bind(ctc_net *net, const float *const *host_params,
                        void *workspace, size_t ws_bytes, int32_t max_batch,
                        void *stream);

/* Kinds of op sequences a network may run as one kernel each (bit mask
 * for ctc_net_set_fusion).  Both keep every stored tensor's arithmetic and
 * roundings; while a kind is on, the internal tensors of its fused
 * sequences are not written (ctc_net_tensor shows stale data), except in
 * passes where an activation fault is armed on one of them: those run the
 * ops separately, so the fault lands as it would without fusion.
 *  CTC_FUSE_IR: (fp16) expand 1x1 + ReLU -> depthwise 3x3 pad 1 + ReLU ->
 *    project 1x1 (+ residual of the block input), the two internal tensors
 *    read by nothing else, with those tensors in LDS; applied to the block
 *    shapes where the fused kernel is the faster one (output maps larger
 *    than 8x8).  Also a block without an expand conv: depthwise 3x3
 *    stride 1 pad 1 (+ ReLU) -> pointwise 1x1 on at most 32 channels, the
 *    depthwise output read by nothing else.  Bit-identical to the separate
 *    kernels.
 *  CTC_FUSE_BLOCK: (fp32) the basic blocks of a residual network (Sec.
 *    IV's ResNets).  Identity blocks of 16, 32 or 64 channels: conv 3x3
 *    stride 1 pad 1 + ReLU -> conv 3x3 stride 1 pad 1 + the first conv's
 *    input + ReLU, the tensor between them read by nothing else; applied to
 *    passes large enough that the fused tiles fill the GPU.  Downsampling
 *    blocks 16 -> 32 and 32 -> 64 channels: conv 3x3 stride 2 pad 1 + ReLU
 *    and a 1x1 stride 2 projection shortcut of the same input, then conv
 *    3x3 stride 1 pad 1 + the shortcut + ReLU, both internal tensors read
 *    once; applied to every pass.  The first conv's output is computed per
 *    output tile (with a one-pixel overlap) and kept in LDS.  Fused blocks
 *    give bit-identical results to their separate kernels.
 *  CTC_FUSE_STEM: (fp16) a 7x7 stride-2 stem conv + ReLU on the 3-channel
 *    input (32 or 64 outputs) and the 3x3 stride-2 pad-1 max pool after it
 *    (ResNet-18), the stem output read by nothing else: the stem outputs
 *    each pooled tile needs are computed into LDS and pooled there;
 *    bit-identical to the two kernels.
 *  CTC_FUSE_POOL: a dense conv whose output only feeds a 2x2 stride-2
 *    max pool (VGG): the pool runs in the conv's epilogue, on spatial
 *    output tiles whose 2x2 windows lie inside the tile, where the conv's
 *    kernel for that shape has the pool (fp16 layers whose tiles waste at
 *    most 1/6 of the work at the map edges); bit-identical to the two
 *    kernels. */
typedef enum {
    CTC_FUSE_IR = 1,
    CTC_FUSE_BLOCK = 2,
    CTC_FUSE_STEM = 4,
    CTC_FUSE_POOL = 8
} ctc_fuse_kind;

/* Selects the fusion kinds in effect (default: all four; 0 runs every op
 * separately).  Errors:
 * CTC_ERR_ARG (NULL net, unknown bits). */
ctc_status ctc_net_set_fusion(ctc_net *net, int32_t kinds);

/* Sets ref and tau used by ctc_network_forward (default: ref 0, tau +Inf,
 * nothing flagged).  Errors: CTC_ERR_ARG (NULL net). */
ctc_status ctc_net_set_threshold(ctc_net *net, float ref, float tau);

typedef enum {
    CTC_REEXEC_NONE = 0,     /* one pass over this batch; flags written,
                                nothing re-run */
    CTC_REEXEC_SYNC = 1,     /* as DEFERRED, then ctc_network_flush before
                                returning (the host waits) */
    CTC_REEXEC_DEFERRED = 2  /* queued: see ctc_network_forward */
} ctc_reexec;

/* Sec. II-B: protected inference of `batch` images.
 *   x_nchw  device [batch][in_c][in_h][in_w] fp32 (read by this call's
 *           stream work only: images are staged on the device at once)
 *   out     device [batch][classes + protect] fp32: logits, then S
 *   flags   device [batch] uint8 (1 = flagged) or NULL
 * Re-execution (Sec. II-B): a flagged image runs once more and its output
 * row in `out` is overwritten; the re-run's own flag is ignored.
 * DEFERRED mode keeps a FIFO queue of inferences: the call appends its
 * images; images flagged by the detector go to the queue's front as soon
 * as that pass's detector result is read (a call reads the results of the
 * pass six back, never waiting for the current one); every pass runs
 * exactly `batch` queued inferences, and a second pass runs once the
 * backlog reaches `batch`.  So re-execution costs about the flagged
 * fraction of a pass and never changes a pass's shape.  A call's output
 * rows are final after later calls have processed them (normally within
 * the next seven) or after ctc_network_flush; `out` and `flags` must stay
 * allocated until then.  The passes of one net must be issued on one
 * stream.
 * Armed activation faults hit the first execution of their image index in
 * every call, never a re-execution (the fault is transient).
 * 0 <= batch <= max_batch.  Errors: CTC_ERR_ARG, CTC_ERR_STATE (not bound),
 * CTC_ERR_DEVICE. */
ctc_status ctc_network_forward(ctc_net *net, int32_t batch,
                               const float *x_nchw, float *out,
                               uint8_t *flags, int32_t reexec, void *stream);

/* Runs every queued inference, including the re-executions their
 * detectors ask for (host waits).  Errors: CTC_ERR_STATE, CTC_ERR_DEVICE. */
ctc_status ctc_network_flush(ctc_net *net, void *stream);

/* ---- HIP graph replay (launch-bound networks) ---------------------------- */

typedef struct ctc_graph ctc_graph;

#define CTC_GRAPH_MAX_IMAGES (1 << 20)

/* Sec. II-B protected inference captured once as a HIP graph, for
 * networks whose passes cost less GPU time than the host takes to issue
 * them.  The graph holds `passes` passes of `batch` images; pass k takes
 * images [k*batch, (k+1)*batch) of x_nchw and writes the same rows of `out`
 * and `flags`, each exactly as ctc_network_forward with CTC_REEXEC_NONE
 * does (detector run, nothing re-run inside the graph).
 *   x_nchw  device [passes*batch][in_c][in_h][in_w] fp32
 *   out     device [passes*batch][classes + protect] fp32: logits, then S
 *   flags   device [passes*batch] uint8 (1 = flagged) or NULL
 * The pointers, pass shapes and the threshold are fixed at capture; the
 * buffers' contents and the net's parameters are read at each replay (so
 * parameter faults injected later are seen).  Capture issues no device
 * work.  The graph owns pinned row tables and a device flag buffer; the net
 * must outlive it.  1 <= batch <= max_batch, passes*batch <=
 * CTC_GRAPH_MAX_IMAGES.  Errors: CTC_ERR_ARG, CTC_ERR_STATE (not bound,
 * per-op profiling on, activation faults armed), CTC_ERR_DEVICE. */
ctc_status ctc_graph_create(ctc_net *net, int32_t batch, int32_t passes,
                            const float *x_nchw, float *out, uint8_t *flags,
                            ctc_graph **graph);

/* Replays the graph on `stream`.  CTC_REEXEC_NONE: enqueues the replay and
 * returns.  CTC_REEXEC_SYNC (protected nets only): waits for the replay,
 * then runs every flagged image once more (Sec. II-B), overwriting its row
 * of `out`, and waits for that; the re-runs' own flags are not kept, so
 * `flags` holds the detector's verdicts.  *n_flagged (may be NULL) receives
 * the number of flagged images (0 with CTC_REEXEC_NONE).  Replays and the
 * net's other passes must be issued on one stream.  Errors: CTC_ERR_ARG,
 * CTC_ERR_STATE (SYNC on an unprotected net), CTC_ERR_DEVICE. */
ctc_status ctc_graph_launch(ctc_graph *graph, int32_t reexec,
                            int32_t *n_flagged, void *stream);

/* Waits for the device, then frees the graph and its tables. */
void ctc_graph_destroy(ctc_graph *graph);

/* ---- fault injection (campaigns, Sec. III-A) ---------------------------- */

typedef enum {
    CTC_SITE_WEIGHT = 0, CTC_SITE_BIAS = 1, CTC_SITE_BN_MEAN = 2,
    CTC_SITE_BN_VAR = 3, CTC_SITE_BN_GAMMA = 4, CTC_SITE_BN_BETA = 5,
    CTC_SITE_ACT = 6
} ctc_site;

typedef struct {
    int32_t site;   /* ctc_site */
    int32_t layer;  /* op index; for CTC_SITE_ACT the tensor id (0 = input,
                       n_ops = the final output logits || S) */
    int64_t index;  /* logical element index: deployed canonical layout
                       (conv KCRS, FC [rows][in] with the classifier's extra
                       row last, bias/BN [c_out]); activations [c][h][w] of
                       one image */
    int32_t bit;    /* bit of the stored representation, 0 = LSB: weights
                       and activations 16 bits in fp16 nets (fp32-stored
                       tensors 32), bias and BN always 32 */
    int32_t image;  /* CTC_SITE_ACT: batch row the flip applies to */
} ctc_fault;

/* Applies n single-bit flips.  Parameter flips change the deployed device
 * parameters at once (a bias/BN flip re-derives that channel's folded
 * scale/shift from the flipped canonical value).  Activation flips are
 * armed: the first execution of image `image` of every later call gets
 * the stored element flipped right after the tensor is produced, until
 * cleared.  Stream-ordered: parameter writes are enqueued on `stream`.
 * Errors: CTC_ERR_ARG (site, index or bit out of range), CTC_ERR_STATE,
 * CTC_ERR_DEVICE. */
ctc_status ctc_inject_bitflip(ctc_net *net, const ctc_fault *faults,
                              int32_t n, void *stream);

/* Undoes every parameter flip (XOR again, in reverse order) and disarms
 * every activation flip.  Stream-ordered like ctc_inject_bitflip.
 * Errors: CTC_ERR_STATE, CTC_ERR_DEVICE. */
ctc_status ctc_clear_faults(ctc_net *net, void *stream);

/* ---- introspection ------------------------------------------------------ */

/* One single-bit fault site of a bound network (Sec. III-A fault model). */
typedef struct {
    int32_t site;      /* ctc_site */
    int32_t layer;     /* op index, or the tensor id for CTC_SITE_ACT */
    int64_t elements;  /* valid ctc_fault.index values are 0 .. elements-1 */
    int32_t bits;      /* valid ctc_fault.bit values are 0 .. bits-1 */
    int32_t pad;
} ctc_site_info;

/* Lists the fault sites of `net`: for every op in order its deployed
 * parameters (weights, then bias, BN mean, var, gamma, beta where
 * present), then, if with_acts, every stored tensor 0 .. n_ops (the last
 * is the final output row, logits || S).  A fault drawn uniformly over
 * sum(elements * bits) is a uniform single-bit fault of the deployed
 * network.  Writes min(total, cap) entries to out (out may be NULL when
 * cap is 0) and the total to *n.  Errors: CTC_ERR_ARG, CTC_ERR_STATE (not
 * bound). */
ctc_status ctc_net_fault_sites(const ctc_net *net, int32_t with_acts,
                               ctc_site_info *out, int32_t cap, int32_t *n);

/* Device address and layout of tensor t (0 .. n_ops-1; the final output is
 * the caller's `out`): NHWC with *c_stored channels (>= logical channels),
 * *dtype the storage type, image stride h*w*c_stored elements. */
ctc_status ctc_net_tensor(const ctc_net *net, int32_t t, void **dev,
                          int32_t *c_stored, int32_t *h, int32_t *w,
                          int32_t *dtype);

/* Device address of deployed weight element `index` of op `layer` (the
 * canonical logical index of ctc_fault, Sec. III-A's fault sites) inside
 * the bound workspace, and its stored width in *bits (16 in fp16 nets, 32
 * else): the element a CTC_SITE_WEIGHT fault with the same (layer, index)
 * flips.  Read-only introspection for tests; the address stays valid
 * while the net is bound.  Errors: CTC_ERR_ARG (NULL pointer, bad layer or
 * index, op without weights), CTC_ERR_STATE (not bound). */
ctc_status ctc_net_weight_address(ctc_net *net, int32_t layer, int64_t index,
                                  void **dev, int32_t *bits);

/* Role the library derived for op i (ctc_role; CTC_ROLE_NONE for non-conv
 * ops or protect = 0). */
int32_t ctc_net_role(const ctc_net *net, int32_t i);

/* ---- measurement support ---------------------------------------------- */

/* While enabled, every stage of every forward pass (slot 0: input staging;
 * slot 1+i: op i; slot n_ops+1: detector) is bracketed by HIP events on the
 * call's stream.  Errors: CTC_ERR_ARG. */
ctc_status ctc_net_profile(ctc_net *net, int32_t enable);

/* Synchronises the timed work, then writes per slot (n_ops + 2 entries)
 * the number of timed launches and their summed duration in milliseconds,
 * and resets the counters.  Errors: CTC_ERR_ARG, CTC_ERR_DEVICE. */
ctc_status ctc_net_profile_read(ctc_net *net, int32_t *launches,
                                double *total_ms);

/* Name of the kernel op i launches for a batch of nimg images (as listed by
 * rocprofv3), copied into name[cap].  Errors: CTC_ERR_ARG. */
ctc_status ctc_net_op_kernel(const ctc_net *net, int32_t i, int32_t nimg,
                             char *name, int32_t cap);

void ctc_net_destroy(ctc_net *net);
const char *ctc_last_error(void);   /* message of this thread's last error */
int32_t ctc_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* CTC_H */
