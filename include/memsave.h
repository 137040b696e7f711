/*
 * memsave.h -- C ABI of the MI355X (gfx950) selective-differentiation layers.
 *
 * The library implements the forward and backward pass of the layers that
 * are linear in both their input and their parameters -- Conv2d, its
 * transpose, Linear and BatchNorm in evaluation mode (Sec. 2.2.1 names the
 * transposed convolution beside the others; App. B lists ConvTransposeNd
 * among the layers it covers) -- driven by a differentiability mask
 * (Sec. 2.2.1 of "Lowering PyTorch's Memory Consumption for Selective
 * Differentiation", arXiv 2404.12406).  The input Jacobian of such a layer
 * needs only the weight, the weight Jacobian needs only the input and the
 * bias Jacobian needs nothing, so a forward call keeps the layer input only
 * when the weight gradient is requested, and a backward call launches only
 * the gradient work whose flag is set.  Selective differentiation -- asking
 * for gradients of a subset of the leaves -- is the problem statement of
 * Sec. 1; the forward/backward pair mirrors the autograd primitive of
 * Sec. 2.2 (a forward that decides what to save, a backward that returns
 * only the needed gradients).
 *
 * Conventions shared by every entry point
 *  - Every buffer is caller-allocated device memory; the library never
 *    frees or copies caller memory.  `ms_tensor.data` is a device pointer.
 *  - Shapes are given in logical PyTorch order, strides in elements.
 *    The kernels read dense channels-last tensors (NHWC activations, KRSC
 *    filters, row-major matrices).  For MS_CONV2D, MS_CONV_TRANSPOSE2D,
 *    MS_LINEAR, MS_BN_EVAL and MS_AVGPOOL any non-negative strides are
 *    accepted (NCHW, strided slices, transposed views, broadcast inputs);
 *    output and gradient buffers must not overlap themselves.  Tensors in
 *    another layout are staged: copied into the kernels' layout in transient
 *    workspace before the launch and back after it, on the same stream
 *    (counted in ms_account.transient_workspace_bytes).  The record still
 *    borrows the caller's own x, never a staged copy.  BN-eval on a plain
 *    NCHW tensor runs in place, without staging.  5-D tensors (the 3-D
 *    kinds) must be channels-last (NDHWC / KTRSC, torch.channels_last_3d);
 *    MS_RELU and MS_DROPOUT take x dense in any order of its dims with y and
 *    the gradients in x's strides; 1-D tensors (biases, BN statistics) are
 *    contiguous.  Anything else returns MS_E_LAYOUT.
 *  - dtypes: MS_F32 or MS_BF16; all tensors of one call share one dtype.
 *    Products are accumulated in fp32 and rounded once to the output dtype
 *    (round to nearest even).
 *  - Every tensor has fewer than 2^31 elements (MS_E_UNSUPPORTED otherwise).
 *  - All work is enqueued on the caller's stream (`stream` is a
 *    hipStream_t; NULL = the null stream); no call synchronises the device
 *    except the first use of a larger transient workspace on a stream.
 *  - Validation runs before any launch.  On error no kernel is launched, no
 *    record is created and the ledger is unchanged; the status says why and
 *    ms_last_error() gives a human-readable detail (thread-local).
 *  - Asynchronous device faults surface as MS_E_HIP from a later call.
 *  - Calls on different streams that overlap on one device are safe: each
 *    stream gets its own transient workspace.
 */
#ifndef MEMSAVE_H
#define MEMSAVE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MS_OK = 0,
    MS_E_NULL = 1,        /* a required pointer is NULL                          */
    MS_E_MASK = 2,        /* mask bits invalid, or grad buffers do not match it  */
    MS_E_SHAPE = 3,       /* shapes inconsistent                                 */
    MS_E_DTYPE = 4,       /* unsupported or mixed dtypes                         */
    MS_E_LAYOUT = 5,      /* strides are not the required memory order           */
    MS_E_UNSUPPORTED = 6, /* valid but not implemented (dilation, size limits)   */
    MS_E_CONSUMED = 7,    /* backward already ran on this record                 */
    MS_E_NOMEM = 8,       /* transient workspace allocation failed               */
    MS_E_HIP = 9,         /* a HIP runtime call or kernel launch failed          */
    MS_E_ARG = 10         /* any other invalid argument                          */
} ms_status;

/* Differentiability mask (requires_grad of the layer's parents). For BN-eval
 * the weight is gamma and the bias is beta. */
enum { MS_RG_INPUT = 1u, MS_RG_WEIGHT = 2u, MS_RG_BIAS = 4u };

typedef enum { MS_F32 = 0, MS_BF16 = 1 } ms_dtype;

/* A device tensor view.  `data` may be NULL only when the tensor has zero
 * elements. */
typedef struct {
    void *data;
    int32_t dtype;       /* ms_dtype */
    int32_t ndim;        /* 1, 2, 4 or 5 */
    int64_t shape[5];
    int64_t stride[5];   /* in elements */
} ms_tensor;

typedef enum {
    MS_CONV2D = 0,       /* y = W * x + b, cross-correlation, zero padding, dilation 1, groups 1
                            x[N,C,H,W], W[K,C,R,S], b[K] or NULL, y[N,K,P,Q],
                            P = (H + 2 pad_h - R) / stride_h + 1 (likewise Q)              */
    MS_LINEAR = 1,       /* y = x W^T + b: x[M,K_in], W[N_out,K_in], b[N_out] or NULL, y[M,N_out] */
    MS_BN_EVAL = 2,      /* y = gamma (x - mean) / sqrt(var + eps) + beta per channel,
                            x[N,C,H,W] or x[N,C]; W = gamma[C], b = beta[C]
                            (both NULL for affine=False); running stats are fixed buffers  */
    MS_AVGPOOL = 3,      /* global average pool x[N,C,H,W] -> y[N,C]; no parameters        */
    MS_RELU = 4,         /* y = max(x, 0) elementwise (NaN and -0 pass through); x dense
                            in any order of its dims, y in the strides of x; no
                            parameters.  Forward through ms_relu_forward() only           */
    MS_CONV_TRANSPOSE2D = 5, /* y = transposed convolution of x (torch.nn.ConvTranspose2d with
                            dilation 1, groups 1): x[N,C_in,H,W], W[C_in,C_out,R,S]
                            (kernel layout: memory [C_in][R][S][C_out]), b[C_out] or NULL,
                            y[N,C_out,H_out,W_out], H_out = (H-1) stride_h - 2 pad_h + R
                            + out_pad_h (likewise W_out), 0 <= out_pad < stride:
                              y[n,o,h',w'] = b[o] + sum of x[n,i,h,w] W[i,o,r,s]
                              over h stride_h - pad_h + r = h', w stride_w - pad_w + s = w'.
                            It is the adjoint of the convolution that maps [N,C_out,H_out,
                            W_out] to [N,C_in,H,W] with filter W, stride and pad: its
                            forward runs that convolution's input-gradient kernel (plus
                            the bias), its input gradient that convolution's forward
                            kernel, its weight gradient that convolution's weight-gradient
                            kernel with x in the role of the output gradient.  The save
                            rule is the convolution's.  A 1-D (transposed) convolution is
                            the 2-D one with H = R = 1, stride_h = 1, pad_h = 0.          */
    MS_DROPOUT = 6,      /* y = x * m / (1 - p), m a random keep mask; layouts as MS_RELU;
                            no parameters.  Forward through ms_dropout_forward() only    */
    MS_CONV3D = 7,       /* 3-D MS_CONV2D (torch.nn.Conv3d, dilation 1, groups 1):
                            x[N,C,D,H,W], W[K,C,T,R,S], b[K] or NULL, y[N,K,Do,P,Q],
                            Do = (D + 2 pad_d - T) / stride_d + 1; channels-last 5-D.
                            Runs the 2-D kernels on the input with its T depth taps
                            folded into the channels (transient workspace of T / stride_d
                            times x in the forward and weight gradient)                  */
    MS_CONV_TRANSPOSE3D = 8 /* 3-D MS_CONV_TRANSPOSE2D: x[N,C_in,D,H,W], W[C_in,C_out,T,R,S],
                            b[C_out] or NULL, y[N,C_out,Do,Ho,Wo], Do = (D-1) stride_d
                            - 2 pad_d + T + out_pad_d; the adjoint of the MS_CONV3D with
                            filter W read as [K = C_in, C = C_out, T, R, S]               */
} ms_kind;

typedef struct {
    int32_t kind;               /* ms_kind */
    int32_t stride[2];          /* conv: stride (h, w), each >= 1 */
    int32_t pad[2];             /* conv: zero padding (h, w), each >= 0 */
    float eps;                  /* BN-eval: epsilon (> 0) */
    const ms_tensor *running_mean;  /* BN-eval: mu_hat[C]; never differentiable */
    const ms_tensor *running_var;   /* BN-eval: sigma_hat^2[C]; never differentiable */
    int32_t out_pad[2];         /* transposed conv: output padding (h, w), 0 <= out_pad < stride;
                                   ignored by the other kinds */
    int32_t stride_d, pad_d, out_pad_d; /* 3-D kinds: the depth axis's stride (>= 1), pad
                                   (>= 0) and output padding (transposed, < stride_d) */
} ms_layer;

/* Opaque saved-tensor record (the AD tape entry of one layer call). */
typedef struct ms_record ms_record;

/* Bits of ms_account.borrowed: which caller tensors a record keeps.
 * MS_SAVED_BITS: a ReLU's 1-bit mask; MS_SAVED_Y (policy accounting only):
 * the layer output, which stock PyTorch's ReLU keeps; MS_SAVED_MASK8 (policy
 * accounting only): the one-byte-per-element mask stock PyTorch's dropout
 * keeps. */
enum { MS_SAVED_X = 1u, MS_SAVED_W = 2u, MS_SAVED_MEAN = 4u, MS_SAVED_VAR = 8u, MS_SAVED_BITS = 16u,
       MS_SAVED_Y = 32u, MS_SAVED_MASK8 = 64u };

/* Bits of ms_account.kernels: what the record's backward will launch. */
enum { MS_K_DGRAD = 1u, MS_K_WGRAD = 2u, MS_K_BGRAD = 4u };

typedef struct {
    uint64_t saved_activation_bytes;  /* bytes of non-parameter tensors kept (the layer input) */
    uint64_t referenced_param_bytes;  /* bytes of parameters / running stats kept by reference */
    uint64_t transient_workspace_bytes; /* workspace the backward needs (released after it)   */
    uint32_t mask;                    /* the mask the record was created with               */
    uint32_t borrowed;                /* MS_SAVED_* bits                                   */
    uint32_t kernels;                 /* MS_K_* bits: backward launch plan                  */
    uint32_t reserved;
} ms_account;

/* Comparison policies of ms_policy_account(). */
enum {
    MS_POLICY_SELECTIVE = 0,       /* the rule of Sec. 2.2.1 (what this library does)      */
    MS_POLICY_PYTORCH_DEFAULT = 1, /* stock PyTorch: conv/BN-eval keep x whenever any flag
                                      is set (Fig. 2, App. B); Linear is already selective */
    MS_POLICY_ALL_TRUE = 2         /* every parent requires grad ("All", Sec. 3)          */
};

/*
 * ms_layer_forward -- y = layer(x; W, b), then record what backward needs.
 *
 * Sec. 2.2.1: with mask bit WEIGHT set the record borrows x (the weight
 * Jacobian needs it); with bit INPUT set it borrows W (the input Jacobian
 * needs it; for BN-eval gamma and running_var); nothing is kept for the
 * bias.  A record borrows: the caller must keep the borrowed tensors alive
 * and unmodified until ms_layer_backward() or ms_record_free().
 * mask == 0 launches the forward only and sets *rec = NULL (no record, as
 * autograd records no node).  Otherwise *rec receives a new record and its
 * saved_activation_bytes are added to the process-wide ledger.
 * x, W, b, y: see ms_kind.  W must be NULL for MS_AVGPOOL; b may be NULL.
 * y is caller-allocated and fully overwritten.  A bf16 convolution whose
 * channel count is not a multiple of 8 uses transient workspace for
 * zero-padded channel copies (MS_E_NOMEM if it cannot be had; nothing is
 * launched then).
 */
ms_status ms_layer_forward(const ms_layer *layer, const ms_tensor *x, const ms_tensor *W,
                           const ms_tensor *b, uint32_t mask, const ms_tensor *y,
                           ms_record **rec, void *stream);

/*
 * ms_relu_mask_bytes -- size of the mask ms_relu_forward() writes for an
 * n-element tensor: 4 * ceil(n / 32) bytes (0 for n <= 0).  Bit i of the
 * mask (bit i % 8 of byte i / 8) belongs to element i in memory order.
 */
uint64_t ms_relu_mask_bytes(int64_t n);

/*
 * ms_relu_forward -- y = max(x, 0), keeping one bit per element for backward.
 *
 * Sec. 2.2.2: an activation that stores its output keeps the next linear
 * layer's input alive whatever that layer's mask, which cancels the saving
 * of Sec. 2.2.1; the input gradient of ReLU needs only which outputs are
 * positive.  The paper's ReLU keeps a one-byte boolean per element and names
 * one-bit booleans as the next step; this one keeps one bit.
 * mask: 0 or MS_RG_INPUT (MS_E_MASK otherwise).  x and y: same shape, dtype
 * and layout (see MS_RELU); y is fully overwritten.  With INPUT set, `bits`
 * is caller-allocated device memory of ms_relu_mask_bytes(numel) bytes,
 * 4-byte aligned (MS_E_ARG otherwise), fully overwritten, and borrowed by
 * *rec (it is the record's saved_activation_bytes) until backward or
 * ms_record_free(); neither x nor y is kept.  With mask 0, bits may be NULL
 * and *rec = NULL.  Backward is ms_layer_backward(rec, grad_y, grad_x, NULL,
 * NULL, stream): grad_x[i] = bit i ? grad_y[i] : 0, where bit i = !(y_i <= 0)
 * (a NaN output passes its gradient, as PyTorch's ReLU does).  ms_layer_forward()
 * rejects MS_RELU (MS_E_ARG).
 */
ms_status ms_relu_forward(const ms_tensor *x, const ms_tensor *y, void *bits, uint32_t mask, ms_record **rec,
                          void *stream);

/*
 * ms_dropout_blocks -- generator blocks one ms_dropout_forward() call over n
 * elements consumes: ceil(n / 4) (0 for n <= 0).  Calls whose offsets are at
 * least this far apart under one seed draw disjoint parts of the stream.
 */
uint64_t ms_dropout_blocks(int64_t n);

/*
 * ms_dropout_forward -- y = x * m / (1 - p), keeping the generator state
 * instead of m for backward.
 *
 * Sec. 2.2.2: a dropout that stores its mask (or its output) keeps
 * activation memory alive for backward whatever the next linear layer's
 * mask says; the paper's dropout keeps the random state and draws the mask
 * again in backward, for some extra compute.  The draw is Philox4x32 with 10
 * rounds (Salmon, Moraes, Dror, Shaw, SC 2011): element i (memory order)
 * takes word i mod 4 of the block with counter (b mod 2^32, b div 2^32, 0,
 * 0), b = offset + floor(i / 4), under key (seed mod 2^32, seed div 2^32),
 * and is kept iff that word is >= floor(p * 2^32).  Kept elements are
 * multiplied by (float)(1 / (1 - p)), dropped ones by 0 (so a dropped Inf or
 * NaN gives NaN, as in PyTorch); p = 1 writes zeros.
 * p: finite, 0 <= p <= 1 (MS_E_ARG otherwise).  mask: 0 or MS_RG_INPUT
 * (MS_E_MASK otherwise).  x and y: same shape, dtype and layout (see
 * MS_RELU); y is fully overwritten.  With INPUT set, *rec keeps (seed,
 * offset, p) and no device memory (saved_activation_bytes = 0); with mask 0,
 * *rec = NULL.  Backward is ms_layer_backward(rec, grad_y, grad_x, NULL,
 * NULL, stream): grad_x = grad_y * m / (1 - p) with m drawn again.
 * ms_layer_forward() rejects MS_DROPOUT (MS_E_ARG).
 */
ms_status ms_dropout_forward(const ms_tensor *x, const ms_tensor *y, float p, uint64_t seed, uint64_t offset,
                             uint32_t mask, ms_record **rec, void *stream);

/*
 * ms_layer_backward -- write exactly the requested gradients for grad_y.
 *
 * grad_x / grad_W / grad_b must be non-NULL exactly for the INPUT / WEIGHT /
 * BIAS bits of the record's mask (MS_E_MASK otherwise), have the shape and
 * dtype of their primal, and are overwritten (not accumulated).  Launches the
 * input-gradient kernel iff INPUT, the weight-gradient contraction iff
 * WEIGHT, the bias-gradient reduction iff BIAS (Sec. 2.2.1).  Consumes the
 * record: its borrowed tensors are released (ledger decremented) and a
 * second call returns MS_E_CONSUMED.  The record itself stays allocated until
 * ms_record_free().
 */
ms_status ms_layer_backward(ms_record *rec, const ms_tensor *grad_y, const ms_tensor *grad_x,
                            const ms_tensor *grad_W, const ms_tensor *grad_b, void *stream);

/*
 * ms_layer_backward_noalloc -- ms_layer_backward() for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Same arguments, checks, kernels,
 * results and record semantics as ms_layer_backward(); the only difference
 * is where the transient workspace (split-K partials, bias-gradient partial
 * rows, transposed or channel-padded copies) lives: in one fixed scratch
 * array of ms_noalloc_scratch_bytes() bytes per GPU, a static device array
 * the library holds on every GPU it runs on until the process ends.  The
 * call allocates nothing (no hipMalloc, hipFree or allocating library
 * routine) and records no profiling events.
 * A backward whose workspace (ms_account.transient_workspace_bytes of the
 * record) exceeds the scratch returns MS_E_UNSUPPORTED before anything is
 * launched; the record is then not consumed and may go to
 * ms_layer_backward() instead.
 * Every call on one GPU uses the same scratch bytes, which keep the last
 * call's contents (no kernel reads scratch it has not written in the same
 * call): calls that may overlap on one GPU -- on different streams, or from
 * several threads without ordering between their streams -- race.  Order
 * them on one stream.
 */
ms_status ms_layer_backward_noalloc(ms_record *rec, const ms_tensor *grad_y, const ms_tensor *grad_x,
                                    const ms_tensor *grad_W, const ms_tensor *grad_b, void *stream);

/* Size in bytes of the fixed scratch of ms_layer_backward_noalloc() (per GPU). */
uint64_t ms_noalloc_scratch_bytes(void);

/* Copy a record's accounting into *out: the bytes of the tensors the
 * forward call kept for the backward (the saved tensors of the autograd
 * primitive, Sec. 2.2) and the transient workspace it used. */
ms_status ms_record_account(const ms_record *rec, ms_account *out);

/* Release a record (and its borrowed bytes if backward did not run): the
 * saved tensors of a graph that is never differentiated are dropped, as
 * Sec. 2.2's primitive frees its context.  NULL is a no-op. */
void ms_record_free(ms_record *rec);

/* Process-wide ledger of borrowed activation bytes: current and peak since
 * the last reset (Sec. 2's proxy for the stored graph is the forward peak). */
ms_status ms_ledger_read(uint64_t *live, uint64_t *peak);
/* Reset the peak to the current live value. */
ms_status ms_ledger_reset(void);

/*
 * ms_policy_account -- the accounting a forward call would produce under
 * `policy` (MS_POLICY_*), without launching anything or touching the ledger.
 * Tensors are validated like ms_layer_forward (data pointers may be NULL).
 * The policies are the comparison of Fig. 2 and App. B: the selective rule
 * of Sec. 2.2.1, stock PyTorch's rule (convolutions and BN-eval keep the
 * input whenever any flag is set; Linear already saves selectively) and the
 * every-parent-differentiable case.  The saved bytes of a forward pass under
 * each policy are what Sec. 2 compares through the forward-peak proxy.
 */
ms_status ms_policy_account(const ms_layer *layer, const ms_tensor *x, const ms_tensor *W,
                            const ms_tensor *b, uint32_t mask, int32_t policy, ms_account *out);

/*
 * Kernel timing (diagnostics).  While armed, the library times every
 * launch of the selected kernel kinds with a pair of HIP events, so the
 * caller can read the kernels' own GPU time over a region of its choice.
 * The bf16 GEMM launches record their pair themselves, stamped at the
 * dispatch's start and end (the kernel alone); the other kernels' pairs are
 * recorded on the launch stream around the launch (they also span its
 * dispatch latency).  A contraction whose output is split over two launches
 * records two pairs.  Only the contraction kernel itself is timed (not the
 * weight transpose or reduction kernels around it).  Kinds name
 * the contraction, not the layer's pass: a transposed convolution's forward
 * is an input-gradient GEMM and its input gradient a forward GEMM.
 *   MS_PROF_FWD   forward convolution / linear GEMM
 *   MS_PROF_DGRAD input-gradient GEMM
 *   MS_PROF_WGRAD weight-gradient GEMM (its split-K partial launch)
 *   MS_PROF_BN    BN-eval forward kernel
 *   MS_PROF_ACT   ReLU and dropout forward and backward kernels
 *   MS_PROF_RED   the reduction passes: a BN-eval backward (its dx-only
 *                 sweep, or its reduction kernel and the finalize kernels
 *                 of dgamma / dbeta, bracketed together) and a bias
 *                 gradient's column sum with its finalize kernel (or the
 *                 finalize alone when the sums rode on the input gradient)
 * ms_profile_start() discards earlier records and arms `kinds` (0 disarms);
 * at most 65536 launches per kind are recorded.  ms_profile_read() waits
 * for the recorded events and returns the number of launches of one kind and
 * their summed duration in milliseconds.  Calls from several threads or
 * streams at once are serialised internally.
 */
enum { MS_PROF_FWD = 1u, MS_PROF_DGRAD = 2u, MS_PROF_WGRAD = 4u, MS_PROF_BN = 8u, MS_PROF_ACT = 16u,
       MS_PROF_RED = 32u };
ms_status ms_profile_start(uint32_t kinds);
ms_status ms_profile_read(uint32_t kind, uint64_t *launches, double *total_ms);

/* Static description of a status code. */
const char *ms_status_str(int32_t status);

/* Detail of the last error on the calling thread ("" if none). */
const char *ms_last_error(void);

/* Library version string. */
const char *ms_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MEMSAVE_H */
