/*
 * dss.h -- exact dense signal scanning on AMD MI355X (gfx950).
 *
 * Evaluates a pooling CNN on every receptive-field-sized window of a 1-D signal
 * or 2-D image at once, with results identical to running the ordinary strided
 * network on each window separately.  The method and its correctness proof are
 * Thom & Gritschneder, "Rapid Exact Signal Scanning with Deep Convolutional
 * Neural Networks": the network is applied in a sliding fashion, every pooling
 * layer is followed by a fragmentation (polyphase reshuffle) of the feature maps,
 * the input is stuffed with dummy samples so that every fragmentation comes out
 * even, and a final defragmentation plus trimming restores the dense output
 * grid (Definition "processing chain", Sect. 4.2; Theorem "processing chain",
 * Sect. 4.3).
 *
 * General conventions
 *  - All functions are C ABI, no C++ exceptions cross it.  Every function that
 *    can fail returns a dss_status; on failure dss_last_error() gives a
 *    human-readable reason for the calling thread.
 *  - Tensors are dense row-major arrays.  Pointers documented as "device" must
 *    be HIP device memory of the current device; "host" pointers are ordinary
 *    memory.  The library never frees caller memory.
 *  - Work on device memory is enqueued asynchronously on the given HIP stream
 *    (0 = the null stream); the caller synchronises.  Argument validation
 *    happens before anything is enqueued: a call that returns an error leaves
 *    every output buffer untouched.
 *  - A 1-D signal is a 2-D one with height 1 (ndim = 1 requires H = 1, filter
 *    heights fh = 1 and pool heights kh = 1).
 *  - Workspaces.  Every evaluation entry point takes device scratch memory as
 *    (workspace, workspace_bytes).  A caller's workspace must hold at least the
 *    bytes the matching geometry query reports and be 256-byte aligned; it is
 *    not read after the call's work completes.  workspace == NULL selects the
 *    plan's own workspace instead (workspace_bytes is then ignored): allocated on
 *    the plan's first request, grown to the largest request seen (growing first
 *    waits for the whole device, then frees and reallocates), freed by
 *    dss_plan_destroy.  Evaluations that pass NULL share that one buffer, so
 *    they must not run concurrently on one plan (on several streams or host
 *    threads); pass a workspace of your own per stream for that.
 *  - Filters use cross-correlation order, as deep-learning frameworks do:
 *    weight[o][i][t_h][t_w] multiplies input sample (y + t_h, x + t_w).  The
 *    paper writes the same operation with a flipped filter (Sect. 3.3); the two
 *    differ only in how the taps are numbered.
 */
#ifndef DSS_H
#define DSS_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum dss_status {
    DSS_OK = 0,
    DSS_E_INVALID = 1,      /* bad argument: NULL pointer, bad descriptor, channel mismatch */
    DSS_E_SHAPE = 2,        /* extents do not fit: signal smaller than the receptive field,
                               fragment extents not divisible by the pool size, too small workspace */
    DSS_E_UNSUPPORTED = 3,  /* valid request outside what the library implements */
    DSS_E_NOMEM = 4,        /* device allocation failed */
    DSS_E_HIP = 5           /* a HIP runtime call or kernel launch failed */
} dss_status;

typedef enum dss_dtype {
    DSS_F32 = 0,            /* IEEE binary32 */
    DSS_BF16 = 1            /* bfloat16: storage type; arithmetic accumulates in binary32 */
} dss_dtype;

typedef enum dss_act {
    DSS_ACT_NONE = 0,
    DSS_ACT_RELU = 1,
    DSS_ACT_TANH = 2
} dss_act;

typedef enum dss_kind {
    DSS_LAYER_CONV = 0,
    DSS_LAYER_MAXPOOL = 1
} dss_kind;

/* One layer of the network as the ordinary (strided, patch-based) CNN sees it.
 *  conv:    multi-channel valid convolution with a filter of fh x fw samples
 *           (Sect. 3.3), then + bias, then the activation.  Fully-connected layers
 *           are convolutions whose filter covers the whole remaining extent.
 *  maxpool: channel-wise maximum over non-overlapping kh x kw blocks starting at
 *           the first sample (Definition "strided function", Sect. 4).
 * A conv directly followed by a maxpool forms one layer of the processing chain;
 * a conv without a pool has k = 1, a pool without a conv before it has the
 * identity transformation (bypass layers, end of Sect. 4.2). */
typedef struct dss_layer {
    int32_t kind;           /* dss_kind */
    int32_t cin, cout;      /* conv: input / output channels */
    int32_t fh, fw;         /* conv: filter extent per axis, >= 1 */
    int32_t act;            /* conv: dss_act */
    int32_t kh, kw;         /* maxpool: block extent per axis, >= 1 */
    const float* weight;    /* conv, host: [cout][cin][fh][fw] binary32 */
    const float* bias;      /* conv, host: [cout] binary32, or NULL for zero bias */
} dss_layer;

/* Geometry of a network applied to an H x W signal (Lemma "processing chain"
 * (a)-(c), Sect. 4.2; stuffing count of Theorem "processing chain", Sect. 4.3),
 * or, for a mixed level ell > 0, of the relaxed/mixed evaluation (appendix:
 * Definition "evalrelaxslide", Lemma "evalrelaxslide", and the operating modes
 * of Theorem "evalrelaxslide"; ell = L is the relaxed evaluation of Definition
 * "evalrelax").  Per axis with N samples, r = rem(N - B + k*_ell, k*_L): if
 * r < k*_ell the last r samples are trimmed first (trimming mode), otherwise
 * k*_L - r dummy samples are stuffed (stuffing mode).  ell = 0 is the dense
 * evaluation: nothing is ever trimmed and the stuffing count is that of
 * Theorem "processing chain". */
typedef struct dss_geometry {
    int32_t ndim;           /* 1 or 2 */
    int32_t in_c, out_c;    /* input channels, output channels of the last layer */
    int32_t n_chain;        /* L: number of processing-chain layers */
    int32_t B_h, B_w;       /* receptive field per axis */
    int32_t K_h, K_w;       /* final stride product k*_L per axis */
    int32_t r_h, r_w;       /* dummy samples stuffed at the end of each axis (stuffing mode) */
    int32_t D_h, D_w;       /* extents the chain runs on: H - trim_h + r_h, W - trim_w + r_w */
    int32_t out_h, out_w;   /* output extents ceil((H - B_h + 1) / step_h), ceil((W - B_w + 1) / step_w);
                               for ell = 0 the dense extents H - B_h + 1, W - B_w + 1 */
    int32_t dtype;          /* dss_dtype of the plan (geometry queries: the dtype passed) */
    int32_t ell;            /* mixed level: chain layers 1..ell run relaxed (strided pooling) */
    int32_t step_h, step_w; /* output sample spacing k*_ell per axis (1 for ell = 0) */
    int32_t trim_h, trim_w; /* samples removed from the end of each axis first (trimming mode) */
    int64_t workspace_bytes;/* device scratch that the evaluation entry points need */
    double conv_flops;      /* algorithmic convolution flops of one evaluation
                               (2 per multiply-add, only the samples the method needs) */
    double pool_bytes;      /* algorithmic bytes of the pooling steps (sliding max-pool + Frag,
                               or strided max-pool for relaxed layers; each tensor read once,
                               written once, at its stored width) */
    double total_bytes;     /* algorithmic bytes of every step (stuff, convs, pools, defrag) */
} dss_geometry;

/* Per-layer geometry for chain layer j (1-based, 1..L), or j = 0 for the
 * trimmed/stuffed input, at a mixed level ell (0 = dense). */
typedef struct dss_layer_geometry {
    int32_t c_h, c_w;       /* dimensionality reduction constant of T_j per axis (1 for identity) */
    int32_t k_h, k_w;       /* pool size k_j per axis (1 when the layer has no pool) */
    int32_t kstar_h, kstar_w;/* stride products k*_j */
    int32_t u_h, u_w;       /* strided extent u_j (Lemma (a)) */
    int32_t U_h, U_w;       /* per-fragment extent after layer j: U_j^row per axis (Lemma (b)) for a
                               sliding layer, W_j (Lemma "evalrelax" (b)) for a relaxed one */
    int32_t F;              /* number of fragments: (k*_j,h / k*_ell,h) * (k*_j,w / k*_ell,w)
                               for a sliding layer (U_j^col, Lemma "evalrelaxslide" (b)), 1 for a
                               relaxed layer and for j = 0 */
    int32_t channels;       /* feature maps after layer j */
    int32_t has_conv, has_pool;
    int32_t relaxed;        /* 1 if 1 <= j <= ell: the layer pools with stride k_j, no Frag */
    int32_t reserved;
} dss_layer_geometry;

typedef struct dss_plan* dss_plan_t;

/* ---------------------------------------------------------------- geometry (host only) */

/* Geometry of `layers` on an H x W signal with `in_channels` channels at mixed
 * level `ell` (0 = dense evaluation, 0..L), without a plan and without touching
 * the GPU.  `dtype` only affects workspace_bytes and the byte counts.
 * DSS_E_SHAPE if H < B_h or W < B_w (the transformation is defined only for
 * signals at least as large as the receptive field); DSS_E_INVALID if ell is
 * outside 0..L. */
dss_status dss_chain_geometry(const dss_layer* layers, int32_t n_layers, int32_t ndim,
                              int32_t in_channels, dss_dtype dtype, int32_t H, int32_t W,
                              int32_t ell, dss_geometry* out);

/* Same for chain layer j (0..L). */
dss_status dss_chain_layer_geometry(const dss_layer* layers, int32_t n_layers, int32_t ndim,
                                    int32_t in_channels, int32_t H, int32_t W, int32_t ell,
                                    int32_t j, dss_layer_geometry* out);

/* ---------------------------------------------------------------- plans */

/* Validates the layer list, derives the processing chain (receptive field B and
 * stride products, Lemma (a)), and copies the weights to the current device in
 * the layouts the kernels read (binary32, or bfloat16 rounded to nearest-even for
 * DSS_BF16 plans; biases stay binary32).  The caller may free `layers` and its
 * weight arrays right after the call.  The plan belongs to the device that was
 * current at creation.  Errors: DSS_E_INVALID (descriptor), DSS_E_UNSUPPORTED
 * (ndim, dtype), DSS_E_NOMEM, DSS_E_HIP. */
dss_status dss_plan_create(const dss_layer* layers, int32_t n_layers, int32_t ndim,
                           int32_t in_channels, dss_dtype dtype, dss_plan_t* out_plan);

/* Releases the plan's device memory (weights and the plan's own workspace).
 * NULL is ignored.  Must not race with an evaluation that is still running on
 * the plan. */
void dss_plan_destroy(dss_plan_t plan);

/* The geometries above for the plan's network (and dtype). */
dss_status dss_plan_geometry(dss_plan_t plan, int32_t H, int32_t W, int32_t ell, dss_geometry* out);
dss_status dss_plan_layer_geometry(dss_plan_t plan, int32_t H, int32_t W, int32_t ell, int32_t j,
                                   dss_layer_geometry* out);

/* ---------------------------------------------------------------- evaluation */

/* Dense evaluation T(signal) = Trim(Defrag_{k*_L}(EvalSlide_L(Stuff(signal))))
 * (Theorem "processing chain", Sect. 4.3), which equals the strided network
 * applied to every window (Slide_{EvalStride_L}).
 *   signal     device, [in_c][H][W] in the plan's dtype (binary32 or bfloat16)
 *   out        device, binary32 [out_c][H - B_h + 1][W - B_w + 1];
 *              out[c][i][j] is channel c of the network's output on the window
 *              whose top-left sample is (i, j)
 *   workspace  device scratch of at least dss_geometry.workspace_bytes bytes
 *              (256-byte aligned), owned by the caller and not read afterwards;
 *              or NULL for the plan's own workspace (see "Workspaces" above)
 *   stream     HIP stream for every launch
 * Concurrent evaluations of one plan are allowed if each uses its own workspace
 * and the plan's timing is off (timed evaluations append to one record list).
 * Errors: DSS_E_INVALID (NULL plan, signal or out; plan of another device),
 * DSS_E_SHAPE (signal smaller than the receptive field, workspace too small),
 * DSS_E_NOMEM (the plan's own workspace could not be allocated), DSS_E_HIP
 * (launch failure). */
dss_status dss_eval_dense(dss_plan_t plan, const void* signal, int32_t H, int32_t W, float* out,
                          void* workspace, int64_t workspace_bytes, hipStream_t stream);

/* Mixed evaluation (appendix: Theorem "evalrelaxslide"; for ell = L Theorem
 * "evalrelax"): chain layers 1..ell are applied in the relaxed fashion (the
 * convolution on the whole signal, then max-pooling with stride k_j and no
 * fragmentation), layers ell+1..L in the sliding fashion with fragmentation,
 * after per-axis trimming or stuffing as described at dss_geometry; the output is
 * defragmented with k*_L / k*_ell and the superfluous samples of the stuffing
 * mode are trimmed.  The result equals dense scanning downsampled by the
 * intermediate stride product: Down_{k*_ell}(Slide_{EvalStride_L}(signal)).
 *   signal     device, [in_c][H][W] in the plan's dtype
 *   ell        mixed level, 0..L (0 gives exactly dss_eval_dense)
 *   out        device, binary32 [out_c][out_h][out_w] with the extents of
 *              dss_plan_geometry(plan, H, W, ell); out[c][i][j] is channel c of the
 *              network's output on the window whose top-left sample is
 *              (step_h * i, step_w * j)
 *   workspace  device scratch of at least dss_geometry.workspace_bytes bytes for
 *              this ell (256-byte aligned), owned by the caller, or NULL for the
 *              plan's own workspace
 * Errors: as dss_eval_dense, and DSS_E_INVALID if ell is outside 0..L. */
dss_status dss_eval_mixed(dss_plan_t plan, const void* signal, int32_t H, int32_t W, int32_t ell,
                          float* out, void* workspace, int64_t workspace_bytes, hipStream_t stream);

/* The intermediate representation after chain layer j (0 <= j <= L; j = 0
 * gives the trimmed/stuffed signal) of the evaluation at mixed level ell
 * (ell = 0: EvalSlide_j(Stuff(signal)); ell > 0: EvalRelaxSlide^ell_j of the
 * trimmed/stuffed signal), as binary32 in the fragment layout [F_j][C_j][U_j,h][U_j,w]
 * (fragment index linearised as for dss_frag; F_j and U_j from
 * dss_plan_layer_geometry).  For a sliding layer j > ell, Lemma "processing
 * chain" (d) (ell = 0) and Lemma "evalrelaxslide" (d) say: with G = k*_j / k*_ell
 * per axis, sample (y, x) of fragment (i mod G_h) * G_w + (w mod G_w) holds, for
 * y = i div G_h + mu_h and x = w div G_w + mu_w, sample (mu_h, mu_w) of the
 * strided network's layer-j output on the window at (k*_ell,h * i, k*_ell,w * w).
 * For a relaxed layer j <= ell (one fragment), Lemma "evalrelaxslide" (c): the
 * u_j-sized block at (i, w) is the layer-j output on the window at
 * (k*_j,h * i, k*_j,w * w).  Same arguments and errors as dss_eval_mixed; `out`
 * must hold F_j * C_j * U_h * U_w floats. */
dss_status dss_eval_slide(dss_plan_t plan, const void* signal, int32_t H, int32_t W, int32_t ell,
                          int32_t j, float* out, void* workspace, int64_t workspace_bytes,
                          hipStream_t stream);

/* ---------------------------------------------------------------- EvalStride baseline */

/* Workspace bytes (and, if conv_flops is not NULL, the algorithmic convolution
 * flops) of dss_eval_stride for a batch of `count` windows, for a layer list
 * (no plan, no GPU) or for a plan.  DSS_E_INVALID if count <= 0. */
dss_status dss_chain_stride_geometry(const dss_layer* layers, int32_t n_layers, int32_t ndim,
                                     int32_t in_channels, dss_dtype dtype, int32_t count,
                                     int64_t* workspace_bytes, double* conv_flops);
dss_status dss_plan_stride_geometry(dss_plan_t plan, int32_t count, int64_t* workspace_bytes,
                                    double* conv_flops);

/* Conventional patch-by-patch scanning, the baseline the method is measured
 * against (EvalStride of Definition "processing chain", Sect. 4.2, applied to
 * each extracted subsignal, Sect. 2.3; the runtime comparison of Sect. 6.3):
 * the windows with row-major indices first .. first+count-1 of the dense output
 * grid are copied out as a batch of B_h x B_w fragments, the strided network
 * runs on every fragment with the same convolution kernels as the dense
 * evaluation (max-pooling with stride k_j, no fragmentation), and each window's
 * output is written to its place in `out`.
 *   signal     device, [in_c][H][W] in the plan's dtype
 *   first      index of the first window, i * (W - B_w + 1) + j for window (i, j)
 *   count      number of windows in this batch (first + count <= number of windows)
 *   out        device, binary32 [out_c][H - B_h + 1][W - B_w + 1] (the layout of
 *              dss_eval_dense); only the batch's positions are written
 *   workspace  device scratch of at least dss_plan_stride_geometry(count) bytes,
 *              256-byte aligned, or NULL for the plan's own workspace
 * Errors: DSS_E_INVALID (NULL pointers, window range, device), DSS_E_SHAPE
 * (signal smaller than the receptive field, workspace too small), DSS_E_HIP. */
dss_status dss_eval_stride(dss_plan_t plan, const void* signal, int32_t H, int32_t W, int64_t first,
                           int32_t count, float* out, void* workspace, int64_t workspace_bytes,
                           hipStream_t stream);

/* ---------------------------------------------------------------- dilated fashion */

/* Extents V_j,h x V_j,w of EvalDilate_j (Lemma "evaldilate" (a):
 * V_j = N - sum_{mu <= j} k*_{mu-1} (c_mu + k_mu - 2) per axis), the workspace
 * dss_eval_dilate needs and its algorithmic convolution flops (all layers), for a
 * layer list (host only) or a plan.  Any output pointer may be NULL.
 * DSS_E_SHAPE if the signal is smaller than the receptive field, DSS_E_INVALID if
 * j is outside 0..L. */
dss_status dss_chain_dilate_geometry(const dss_layer* layers, int32_t n_layers, int32_t ndim,
                                     int32_t in_channels, dss_dtype dtype, int32_t H, int32_t W,
                                     int32_t j, int32_t* V_h, int32_t* V_w, int64_t* workspace_bytes,
                                     double* conv_flops);
dss_status dss_plan_dilate_geometry(dss_plan_t plan, int32_t H, int32_t W, int32_t j, int32_t* V_h,
                                    int32_t* V_w, int64_t* workspace_bytes, double* conv_flops);

/* The network applied in the dilated fashion (appendix: Definition "evaldilate"):
 * layer j applies its convolution and its max-pool to the whole signal with the
 * taps k*_{j-1} samples apart (Definition "dilate"), with no stuffing,
 * fragmentation or trimming; the intermediate EvalDilate_j for j = 0..L is
 * returned.  By Lemma "evaldilate" (d) the strided network's layer-j output on
 * the window at (i, w) is the u_j,h x u_j,w block of samples
 * (i + k*_j,h a, w + k*_j,w b) of EvalDilate_j; for j = L this is the dense
 * output itself, element for element the result of dss_eval_dense.
 *   signal     device, [in_c][H][W] in the plan's dtype
 *   out        device, binary32 [C_j][V_j,h][V_j,w] (for j = L: [out_c][H - B_h + 1][W - B_w + 1])
 *   workspace  device scratch of at least the bytes dss_plan_dilate_geometry gives
 *              (256-byte aligned), or NULL for the plan's own workspace
 * Errors: as dss_eval_dense, and DSS_E_INVALID if j is outside 0..L. */
dss_status dss_eval_dilate(dss_plan_t plan, const void* signal, int32_t H, int32_t W, int32_t j,
                           float* out, void* workspace, int64_t workspace_bytes, hipStream_t stream);

/* ---------------------------------------------------------------- backward (binary32 plans) */

/* Workspace bytes, number of weight-gradient and bias-gradient floats, and the
 * algorithmic convolution flops (forward + weight gradient + input gradient) of
 * dss_backward_dense on an H x W signal, for a layer list (host only) or a plan.
 * with_signal_grad: nonzero if the gradient with respect to the signal is wanted
 * (it adds the first layer's input-gradient convolution).  The workspace
 * depends on the kernels chosen for the input gradients (a zero-bordered copy
 * of the gradient only for those that run on the direct kernel): the plan form
 * is exact for its plan, the layer-list form assumes the choice a plan created
 * at the same time would make.  Output pointers may be NULL.  Errors as
 * dss_chain_geometry. */
dss_status dss_chain_backward_geometry(const dss_layer* layers, int32_t n_layers, int32_t ndim,
                                       int32_t in_channels, int32_t H, int32_t W,
                                       int32_t with_signal_grad, int64_t* workspace_bytes,
                                       int64_t* weight_grad_floats, int64_t* bias_grad_floats,
                                       double* flops);
dss_status dss_plan_backward_geometry(dss_plan_t plan, int32_t H, int32_t W, int32_t with_signal_grad,
                                      int64_t* workspace_bytes, int64_t* weight_grad_floats,
                                      int64_t* bias_grad_floats, double* flops);

/* Gradients of l = sum(grad_out * T(signal)) for the dense evaluation T of
 * dss_eval_dense, for fine-tuning on whole signals (the transformed network is
 * the same function as the strided one on every window; Sect. 6.2 notes that
 * Stuff and Trim have trivial gradients, Frag and Defrag are inverse
 * permutations, and the sliding max-pool needs elementary calculus only).  The
 * call runs the dense forward pass itself, keeping every layer's output in the
 * workspace, then backpropagates through Trim, Defrag, each layer's sliding
 * max-pool + Frag (the gradient of a window's maximum goes to its first maximal
 * sample in row-major order), activation and convolution, and Stuff.  The result
 * equals the sum over all windows of the strided network's gradients.
 *   signal       device, [in_c][H][W] binary32
 *   grad_out     device, binary32 [out_c][H - B_h + 1][W - B_w + 1]
 *   grad_weight  device, binary32: the convolutions in descriptor order, each
 *                [cout][cin][fh][fw] (cross-correlation order, like the weights),
 *                concatenated; written, not accumulated
 *   grad_bias    device, binary32: each convolution's [cout], concatenated
 *   grad_signal  device, binary32 [in_c][H][W], or NULL to skip it
 *   workspace    device scratch of dss_plan_backward_geometry bytes (256-byte aligned),
 *                or NULL for the plan's own workspace
 * Errors: DSS_E_UNSUPPORTED for bfloat16 plans; otherwise as dss_eval_dense. */
dss_status dss_backward_dense(dss_plan_t plan, const void* signal, int32_t H, int32_t W,
                              const float* grad_out, float* grad_weight, float* grad_bias,
                              float* grad_signal, void* workspace, int64_t workspace_bytes,
                              hipStream_t stream);

/* ---------------------------------------------------------------- allocation-free evaluation */

/* Bytes of the fixed workspace of dss_eval_dense_noalloc. */
#define DSS_NOALLOC_SCRATCH_BYTES (64ll * 1024 * 1024)

/* dss_eval_dense for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same evaluation and kernels, bit for bit the same output, with the
 * workspace in a fixed device array of the library (DSS_NOALLOC_SCRATCH_BYTES,
 * held by every device the library runs on until the process ends) instead of
 * a caller or plan buffer.  No device memory is allocated or freed and no HIP
 * event is created: the plan's timing records nothing for these calls.
 *   signal, H, W, out, stream  as for dss_eval_dense
 * All calls on one device share that device's array and leave their data in
 * it: calls that overlap on one device (several streams or host threads) race
 * and must be serialised by the caller.
 * Errors: as dss_eval_dense, and DSS_E_UNSUPPORTED if the signal needs more
 * workspace than DSS_NOALLOC_SCRATCH_BYTES (nothing is enqueued then). */
dss_status dss_eval_dense_noalloc(dss_plan_t plan, const void* signal, int32_t H, int32_t W, float* out,
                                  hipStream_t stream);

/* ---------------------------------------------------------------- Frag / Defrag */

/* Fragmentation Frag_k per axis (Definition "fragmentation" and Lemma
 * "frag-ops", Sect. 4.1) on a planar fragment tensor:
 *   in   device, [S_h*S_w][C][H][W]       (S_h x S_w fragments, row-major)
 *   out  device, [(k_h*S_h)*(k_w*S_w)][C][H/k_h][W/k_w]
 *   out[(a_h*S_h + b_h)*(k_w*S_w) + a_w*S_w + b_w][c][m][n]
 *        = in[b_h*S_w + b_w][c][m*k_h + a_h][n*k_w + a_w]
 * i.e. per axis, sample m*k + a of input fragment b goes to sample m of output
 * fragment a*S + b.  A pure permutation: bit-exact for either element width.
 * DSS_E_SHAPE unless k_h divides H and k_w divides W.  in and out must not overlap. */
dss_status dss_frag(int32_t k_h, int32_t k_w, int32_t S_h, int32_t S_w, int32_t C, int32_t H,
                    int32_t W, dss_dtype dtype, const void* in, void* out, hipStream_t stream);

/* Defragmentation Defrag_k per axis, the inverse of dss_frag (Lemma
 * "defrag-ops", Sect. 4.1, and its simplified form in the appendix):
 *   in   device, [(k_h*S_h)*(k_w*S_w)][C][H][W]
 *   out  device, [S_h*S_w][C][H*k_h][W*k_w]
 *   out[b_h*S_w + b_w][c][y][x]
 *        = in[((y mod k_h)*S_h + b_h)*(k_w*S_w) + (x mod k_w)*S_w + b_w][c][y div k_h][x div k_w] */
dss_status dss_defrag(int32_t k_h, int32_t k_w, int32_t S_h, int32_t S_w, int32_t C, int32_t H,
                      int32_t W, dss_dtype dtype, const void* in, void* out, hipStream_t stream);

/* ---------------------------------------------------------------- telemetry */

/* Per-launch record of an evaluation on a plan with timing enabled. */
typedef struct dss_launch_record {
    const char* kernel;     /* static string: kernel family and variant */
    int32_t chain_layer;    /* 1..L, 0 for stuffing, L+1 for defragmentation */
    int32_t tile_mode;      /* convolutions on the MFMA kernel: 0 spatial tiles of one fragment,
                               1 flat tiles (the fragment batch read as one sequence of samples),
                               2 dilated tiles (one phase of one signal); -1 for every other launch */
    double ms;              /* device time between HIP events around the launch */
    double flops;           /* algorithmic flops of the launch (0 for data movement) */
    double bytes;           /* algorithmic bytes of the launch (each tensor once) */
} dss_launch_record;

/* Enables (1) or disables (0) HIP-event timing of every launch of later
 * evaluations of this plan, and discards the records collected so far (after
 * waiting for their events).  Timing adds two event records per launch on the
 * evaluation stream and is off by default.  Records accumulate over all timed
 * evaluations until the next call of this function; timed evaluations of one
 * plan must not run concurrently from several host threads. */
dss_status dss_plan_set_timing(dss_plan_t plan, int32_t enable);

/* Waits for the events of the collected records and copies up to `cap` of
 * them, oldest first; *count receives the number collected.  Not safe to call
 * concurrently with an evaluation of the same plan. */
dss_status dss_plan_timings(dss_plan_t plan, dss_launch_record* records, int32_t cap, int32_t* count);

/* ---------------------------------------------------------------- misc */

const char* dss_status_string(dss_status s);
/* Reason for the calling thread's last failure ("" if none).  Valid until the
 * thread's next failing call. */
const char* dss_last_error(void);
/* Library version as "major.minor.patch". */
const char* dss_version(void);

#ifdef __cplusplus
}
#endif
#endif /* DSS_H */
