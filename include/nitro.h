/*
 * nitro.h -- C ABI of the MI355X (gfx950) library for the hot path of NITRO-D integer-only
 * training (Pirillo, Colombo, Roveri, "NITRO-D: Native Integer-only Training of Deep
 * Convolutional Neural Networks", arXiv 2407.11698).
 *
 * What the library computes, per integer local-loss block (section 3.2):
 *   forward layers  IntConv2D 3x3 / IntLinear (section 3.2.1, Tab. 1: stride 1, zero padding 1,
 *                   no bias) -> NITRO-Scaling z* = floor(z / SF), SF = 2^8 * fan_in (Eq. 1 and
 *                   the scaling-factor rule of section 3.2.1) -> NITRO-ReLU (section 3.2.2)
 *                   -> optional 2x2/2 max-pool after the last layer (Tab. 1);
 *   learning layer  IntLinear(d -> G) + NITRO-Scaling on the block output (section 3.2, the
 *                   training procedure of section 3.3), RSS loss gradient yhat - y with the
 *                   32-valued one-hot target (Eq. 4; section 3.3.4, Appendix A);
 *   backward        delta^fw = grad * W^il (section 3.3.4) routed back through pool, NITRO-ReLU
 *                   and the forward layers of the block only; int64 weight gradients;
 *   IntegerSGD      Alg. 1, with gamma^fw = AF * gamma, AF = 2^6 * G (Eq. 6).
 * Everything is integer arithmetic; results are bit-exact.
 *
 * Readings of passages the paper leaves open (the same ones the test-side checker uses):
 *   - division rounds toward minus infinity (the paper's floor macro) unless NITRO_ROUND_TRUNC
 *     is chosen, which rounds every division of the step toward zero;
 *   - the NITRO-ReLU mean is (s1 + s2 + 63 + 127) / 4 with s1 = -127/alpha_inv and
 *     s2 = -127/(2 alpha_inv), every division by the chosen rounding;
 *   - the NITRO-ReLU backward is the derivative of its piecewise map at z*: identity for
 *     0 <= z* <= 127, division by alpha_inv for -127 <= z* < 0, zero where the map saturates
 *     (NITRO-Scaling itself passes gradients unchanged, section 3.2.1);
 *   - the loss gradient is per sample; max-pool routes the gradient to the first maximum of the
 *     2x2 window in row-major order; delta^fw uses the learning weights from before the update;
 *   - every layer (learning and output layers included) is rescaled by 2^8 times its own fan-in;
 *     learning and output layers have no NITRO-ReLU.
 *
 * Conventions
 *   - Tensor arguments are DEVICE pointers owned by the caller. The library never frees them and
 *     keeps no reference to them after the work it enqueued has run.
 *   - Layouts: images NHWC (channels innermost); conv weights KRSC [C_out][3][3][C_in];
 *     linear weights [out][in]; the learning layer's input index d runs over the block output in
 *     (h, w, c) order. Activations are int8, weights int32, weight gradients int64,
 *     predictions and gradients int32.
 *   - Every call validates its arguments on the host and returns NITRO_EINVAL before enqueuing
 *     anything when they are wrong. Work is then enqueued asynchronously on the context's stream.
 *   - Data-dependent errors are sticky device flags, read and cleared by nitro_sync_status():
 *     NITRO_EOVERFLOW when a value does not fit its int32 destination (or a weight or gradient
 *     operand exceeds what the kernels can represent), NITRO_ELABEL when a label is outside
 *     [0, G). A kernel that raises a flag still writes its outputs (then unspecified).
 *   - A context is used by one host thread at a time. Calls that overlap on one stream are
 *     ordered by the stream.
 */
#ifndef NITRO_H
#define NITRO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    NITRO_OK = 0,
    NITRO_EINVAL = -1,        /* bad argument: null pointer, zero divisor, bad shape ...     */
    NITRO_EOVERFLOW = -2,     /* a result does not fit its declared integer type             */
    NITRO_ELABEL = -3,        /* a label outside [0, G)                                       */
    NITRO_EHIP = -4,          /* a HIP runtime call failed                                    */
    NITRO_ENOMEM = -5,        /* a device allocation failed                                   */
    NITRO_EUNSUPPORTED = -6   /* valid but not supported by the library (e.g. too many blocks) */
} nitro_status;

typedef enum { NITRO_ROUND_FLOOR = 0, NITRO_ROUND_TRUNC = 1 } nitro_round;
typedef enum { NITRO_CONV3X3 = 0, NITRO_LINEAR = 1 } nitro_layer_kind;

#define NITRO_MAX_LAYERS 4
#define NITRO_MAX_BLOCKS 16

typedef struct nitro_ctx nitro_ctx;

/* Create a context on HIP device `device` that enqueues on `hip_stream` (a hipStream_t; NULL
 * means the null stream). Allocates a few bytes of device memory for the status flags. */
nitro_status nitro_create(nitro_ctx **out, int device, void *hip_stream);
/* Destroy a context (synchronises its stream first). NULL is ignored. */
void nitro_destroy(nitro_ctx *ctx);
/* Change the stream later calls enqueue on. */
nitro_status nitro_set_stream(nitro_ctx *ctx, void *hip_stream);
/* Tile of the tiled int8 MFMA convolution kernels (forward and input gradient): 0 chooses by
 * shape (the default), 128 or 256 output pixels per workgroup force that tile wherever its
 * geometry fits the layer (other layers keep the automatic choice). Results do not depend on it.
 * EINVAL for any other value. */
nitro_status nitro_set_conv_tile(nitro_ctx *ctx, int32_t pixels);
/* Workgroups of the tiled convolution kernels with the 256-pixel tile: 0 chooses by size (the
 * default: for a launch of at least 4 tiles per compute unit, one persistent workgroup per compute
 * unit, each taking tiles b, b + G, b + 2G, ...; otherwise one workgroup per tile), 1 makes every
 * such launch persistent (with about 4 tiles per workgroup), -1 none. Results do not depend on
 * it. EINVAL for any other value. */
nitro_status nitro_set_conv_persistent(nitro_ctx *ctx, int32_t mode);
/* Number of auxiliary streams nitro_train_step runs the blocks' local training on (0 to 3,
 * default 3): the forward pass runs on the context's stream; block b's local training starts
 * when block b's forward is done, on auxiliary stream b mod n, except the last block's, which
 * follows on the context's stream; with 0 everything runs on the context's stream, in that
 * order. The streams are the context's own, created on first use. Results do not depend on it.
 * EINVAL outside 0..3. */
nitro_status nitro_set_aux_streams(nitro_ctx *ctx, int32_t n);
/* Synchronise the stream, then return and clear the sticky device flags: NITRO_OK, or the first
 * of NITRO_EOVERFLOW, NITRO_ELABEL that was raised. */
nitro_status nitro_sync_status(nitro_ctx *ctx);
/* Static description of a status code. */
const char *nitro_status_str(nitro_status s);

/* ------------------------------------------------------------------------------------------ */
/* One integer local-loss block                                                               */
/* ------------------------------------------------------------------------------------------ */

typedef struct {
    int32_t kind;      /* nitro_layer_kind                                                  */
    int32_t c_in;      /* conv: input channels; linear: input features                      */
    int32_t c_out;     /* conv: output channels; linear: output features                    */
} nitro_layer;

typedef struct {
    int32_t n, h, w;                       /* batch; input height and width (1, 1 for linear)  */
    int32_t n_layers;                      /* 1..NITRO_MAX_LAYERS forward layers               */
    nitro_layer layer[NITRO_MAX_LAYERS];   /* all conv or all linear; c_in[j] = c_out[j-1]     */
    int32_t maxpool;                       /* 1: 2x2/2 max-pool after the last NITRO-ReLU      */
    int32_t n_classes;                     /* G of the learning layer; 0: no learning layer,
                                              the caller supplies the output gradient          */
    int32_t alpha_inv;                     /* NITRO-ReLU inverse slope, >= 2                    */
    int32_t round;                         /* nitro_round                                       */
    int32_t d_lr;                          /* learning-layer input of a conv block: 0 reads the
                                              block output; > 0 reads it max-pooled to at most
                                              d_lr features (d^lr of Tab. 6): non-overlapping
                                              kh x kw windows, kh and kw doubled in turn (kh
                                              first) while c (h/kh) (w/kw) > d_lr and a side
                                              can still be halved; the first maximum of a
                                              window (row-major) wins and takes the gradient.
                                              Ignored for linear blocks                          */
} nitro_block_desc;

typedef struct {
    const int32_t *w[NITRO_MAX_LAYERS];    /* forward-layer weights                            */
    const int32_t *w_lr;                   /* learning layer [G][d]; NULL iff n_classes == 0    */
} nitro_block_params;

typedef struct {
    int64_t *dw[NITRO_MAX_LAYERS];         /* weight gradients of the forward layers (required) */
    int64_t *dw_lr;                        /* learning-layer gradient [G][d] (if n_classes > 0) */
} nitro_block_grads;

/* Optional extra outputs of the backward pass; every pointer may be NULL. */
typedef struct {
    int32_t *yhat;                         /* [n][G] learning-layer prediction                 */
    int32_t *e;                            /* [n][G] loss gradient yhat - y                     */
    int32_t *delta;                        /* delta^fw at the learning layer's input: the block
                                              output (pooled), NHWC, or with d_lr its learning
                                              pooling [n][h/kh][w/kw][c]                         */
    int32_t *g[NITRO_MAX_LAYERS];          /* gradient at layer j's pre-activation z_j, NHWC   */
    int64_t *dx;                           /* input gradient of the first layer, NHWC; int64
                                              since no gradient leaves a block in the method,
                                              so nothing bounds it to int32                    */
} nitro_block_taps;

/* Size in bytes of the block's state buffer: what the forward pass saves for the backward pass
 * plus the backward pass's scratch. The caller allocates it (any device allocation, 256-byte
 * aligned) and passes the same buffer to nitro_block_forward and nitro_block_backward. */
nitro_status nitro_block_query(const nitro_block_desc *desc, size_t *state_bytes);

/* Device pointers, inside a block state buffer, of what the forward pass saved for forward layer
 * j: its int8 NHWC output activations (*act; NULL for the last layer, whose output is the
 * caller's a_out) and its NITRO-ReLU region codes (*code; one uint8 per output element: 0 for
 * 0 <= z* <= 127, 1 for -127 <= z* < 0, 2 where the map saturates; for a pooled last layer, one
 * per pooled element: argmax index in the 2x2 window | region << 2). For inspection. */
nitro_status nitro_block_saved(const nitro_block_desc *desc, void *state, int32_t j,
                               int8_t **act, uint8_t **code);

/* Forward layers of one block (section 3.2; training procedure of section 3.3).
 *   x      int8 NHWC [n][h][w][c_in] (or [n][c_in] for linear blocks); must stay unchanged
 *          until the matching nitro_block_backward has run;
 *   a_out  int8 NHWC block output, [n][h/2][w/2][c_out] when maxpool, else [n][h][w][c_out];
 *   state  the block's state buffer (nitro_block_query). */
nitro_status nitro_block_forward(nitro_ctx *ctx, const nitro_block_desc *desc,
                                 const nitro_block_params *params, const int8_t *x,
                                 int8_t *a_out, void *state);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation): nitro_block_forward without the caller's state
 * buffer. Computes the same a_out (forward layers, NITRO-Scaling, NITRO-ReLU, pool; section 3.2).
 * Everything else the forward pass writes (inner activations, region codes, weight limb planes,
 * max slots, a channel-padded input, the split-K partial sums and padded input rows of linear
 * layers on the int8 MFMA GEMM) goes to a library-owned device array of 64 MiB per device,
 * allocated with the library's code and held until the process ends; the call allocates and
 * frees nothing. Nothing in that array is meant for the caller, and no nitro_block_backward can
 * follow from it. NITRO_EUNSUPPORTED when the block needs more than 64 MiB of it (the forward
 * part of nitro_block_query's state: about 2 bytes per inner and last-layer activation plus the
 * weight planes, and for linear layers 8 bytes per output per K split), NITRO_EHIP if the
 * array's device address could not be found when the context was created. Every call on a
 * device shares that device's array: calls that overlap on one device (other streams or
 * contexts) race on it; calls ordered on one stream do not. */
nitro_status nitro_block_forward_noalloc(nitro_ctx *ctx, const nitro_block_desc *desc,
                                         const nitro_block_params *params, const int8_t *x,
                                         int8_t *a_out);

/* Local training of one block, with the weights from before any update (section 3.3):
 * learning layer -> yhat, loss gradient e = yhat - 32*onehot(labels), dW^il = e^T a_out,
 * delta^fw = e W^il, then back through pool, NITRO-ReLU and the forward layers: dW per layer.
 *   x, a_out  the same buffers as the forward call;
 *   labels    int32 [n] in [0, G) (NITRO_ELABEL otherwise); used iff n_classes > 0;
 *   delta_out int32 gradient at the block output, same shape as a_out; used iff n_classes == 0;
 *   grads     int64 outputs (overwritten);
 *   taps      optional extra outputs (may be NULL). */
nitro_status nitro_block_backward(nitro_ctx *ctx, const nitro_block_desc *desc,
                                  const nitro_block_params *params, const int8_t *x,
                                  const int8_t *a_out, const int32_t *labels,
                                  const int32_t *delta_out, void *state,
                                  const nitro_block_grads *grads, const nitro_block_taps *taps);

/* ------------------------------------------------------------------------------------------ */
/* One forward layer (thin wrappers over a one-layer block with no pooling and no learning     */
/* layer: the single-layer workload and unit tests)                                             */
/* ------------------------------------------------------------------------------------------ */

typedef struct {
    int32_t n, h, w;       /* batch; input height and width (1, 1 for linear)                  */
    nitro_layer layer;     /* IntConv2D 3x3 (stride 1, zero padding 1) or IntLinear            */
    int32_t alpha_inv;     /* NITRO-ReLU inverse slope, >= 2                                    */
    int32_t round;         /* nitro_round                                                       */
} nitro_layer_desc;

/* Size in bytes of the layer's state buffer (as nitro_block_query for the one-layer block). */
nitro_status nitro_layer_query(const nitro_layer_desc *desc, size_t *state_bytes);

/* The layer's forward pass with NITRO-Scaling (SF = 2^8 fan-in, section 3.2.1) and NITRO-ReLU
 * (section 3.2.2): w int32 (conv KRSC [c_out][3][3][c_in], linear [c_out][c_in]), x int8 NHWC,
 * a_out int8 NHWC [n][h][w][c_out]; x stays unchanged until the matching backward call. */
nitro_status nitro_layer_forward(nitro_ctx *ctx, const nitro_layer_desc *desc, const int32_t *w,
                                 const int8_t *x, int8_t *a_out, void *state);

/* The layer's backward pass from delta, the int32 gradient at its NITRO-ReLU output (shape of
 * a_out): g = the gradient at z through NITRO-ReLU (section 3.2.2; written to g when not NULL),
 * dw = the weight gradient (int64, overwritten; section 3.2.1), and, when dx is not NULL, the
 * int64 gradient at x. EINVAL for a null w, x, a_out, delta, state or dw. */
nitro_status nitro_layer_backward(nitro_ctx *ctx, const nitro_layer_desc *desc, const int32_t *w,
                                  const int8_t *x, const int8_t *a_out, const int32_t *delta,
                                  void *state, int64_t *dw, int32_t *g, int64_t *dx);

/* Output layer on f [n][d] int8: yhat = floor(f W^T / (2^8 d)), e = yhat - 32*onehot(labels),
 * dW = e^T f (int64 [G][d]) -- the global loss gradient of section 3.3. yhat, e may be NULL. */
nitro_status nitro_head_backward(nitro_ctx *ctx, int32_t n, int32_t d, int32_t n_classes,
                                 const int8_t *f, const int32_t *w, const int32_t *labels,
                                 int32_t round, int64_t *dw, int32_t *yhat, int32_t *e);

/* IntegerSGD with weight decay (Alg. 1) on `count` int32 weights, in place:
 *   w' = w - (dw / gamma_inv + [eta != 0] * w / eta),
 * with eta = gamma_inv * lambda_inv (or eta_override when >= 0) and every division rounded per
 * `round`.
 * gamma_inv >= 1, lambda_inv >= 0 (EINVAL otherwise). A result outside int32 raises
 * NITRO_EOVERFLOW (the weight is then left unchanged). */
nitro_status nitro_integer_sgd_step(nitro_ctx *ctx, int32_t *w, const int64_t *dw, int64_t count,
                                    int64_t gamma_inv, int64_t lambda_inv, int64_t eta_override,
                                    int32_t round);

/* Writable weights of one block, for its IntegerSGD step. */
typedef struct {
    int32_t *w[NITRO_MAX_LAYERS];          /* forward-layer weights                            */
    int32_t *w_lr;                         /* learning layer [G][d]; NULL iff n_classes == 0    */
} nitro_block_weights;

/* Hyper-parameters of IntegerSGD (Alg. 1) and of the amplification factor (Eq. 6) for a block or
 * a whole network. */
typedef struct {
    int64_t gamma_inv;        /* gamma_inv of learning and output layers (>= 1)                 */
    int64_t lambda_inv_fw;    /* lambda_inv of forward layers (>= 0, 0: no decay)               */
    int64_t lambda_inv_lr;    /* lambda_inv of learning and output layers                       */
    int64_t af;               /* amplification factor; 0 means 2^6 * G (Eq. 6)                 */
    int64_t eta_fw;           /* < 0: eta = (AF * gamma_inv) * lambda_inv_fw; else this eta     */
    int64_t eta_lr;           /* < 0: eta = gamma_inv * lambda_inv_lr; else this eta           */
    uint64_t dropout_seed;    /* key of the dropout generator (nitro_train_step)               */
    int64_t dropout_step;     /* its step counter: a different value for every iteration        */
    int32_t af_classes;       /* G entering AF = 2^6 G when af == 0 and the block has no
                                 learning layer (n_classes == 0); ignored otherwise             */
    int32_t dropout_conv_ppm; /* dropout rate p_c of conv blocks' outputs, parts per million    */
    int32_t dropout_lin_ppm;  /* dropout rate p_l of linear blocks' outputs (Tab. 6)            */
    int32_t reserved;         /* must be 0                                                      */
} nitro_hparams;

/* IntegerSGD (Alg. 1) of one block after nitro_block_backward: every forward layer with
 * gamma^fw = AF * gamma_inv (Eq. 6), lambda_inv_fw, and the learning layer (when
 * n_classes > 0) with gamma_inv, lambda_inv_lr; one launch. AF = hp->af, or 2^6 G with G the
 * block's n_classes (hp->af_classes for a block without learning layer; EINVAL if both are 0).
 * Weights are updated in place; a result outside int32 raises NITRO_EOVERFLOW and leaves that
 * weight unchanged. EINVAL for a null pointer or a divisor out of range (as
 * nitro_integer_sgd_step) or an eta = gamma * lambda beyond int64. */
nitro_status nitro_block_sgd_step(nitro_ctx *ctx, const nitro_block_desc *desc,
                                  const nitro_block_weights *weights,
                                  const nitro_block_grads *grads, const nitro_hparams *hp);

/* ------------------------------------------------------------------------------------------ */
/* Integer pre-processing of the input data (Appendix A)                                      */
/* ------------------------------------------------------------------------------------------ */

/* Size in bytes of the device workspace nitro_preprocess needs for `count` elements (at most
 * about 1 MiB). EINVAL for count < 1 or count > 2^40. */
nitro_status nitro_preprocess_query(int64_t count, size_t *workspace_bytes);

/* Integer-only normalisation of a whole dataset of unsigned bytes (Appendix A):
 *   mu = sum_i x_i / N,  omega = sum_i |x_i - mu| / N,  out_i = (x_i - mu) * 51 / omega,
 * over all N = count elements, every division rounded per `round`. Readings: mu and omega are
 * single numbers for the dataset; an omega that rounds to 0 is replaced by 1; out is int8, so a
 * value outside [-127, 127] is clamped to it.
 *   x          device, count bytes (any alignment);
 *   out        device, count int8 (may be x itself: normalisation in place);
 *   stats      device, 3 int64 written: mu, the omega divided by, the number of clamped values;
 *   workspace  device, nitro_preprocess_query bytes, any contents (overwritten).
 * Asynchronous on the context's stream; EINVAL for a null pointer, a bad count or rounding. */
nitro_status nitro_preprocess(nitro_ctx *ctx, const uint8_t *x, int64_t count, int32_t round,
                              int8_t *out, int64_t *stats, void *workspace);

/* ------------------------------------------------------------------------------------------ */
/* A whole network: one training iteration                                                    */
/* ------------------------------------------------------------------------------------------ */

typedef struct {
    int32_t n_blocks;                          /* 1..NITRO_MAX_BLOCKS                           */
    nitro_block_desc block[NITRO_MAX_BLOCKS];  /* shapes must chain: block b+1 reads block b's
                                                  output (a linear block after a conv block
                                                  reads it flattened in (h, w, c) order, c_in =
                                                  h w c); every block has n_classes = G > 0    */
    int32_t head;                              /* 1: output layer IntLinear(d_L -> G)           */
} nitro_net_desc;

typedef struct {
    int32_t *w[NITRO_MAX_BLOCKS][NITRO_MAX_LAYERS];   /* forward-layer weights (updated)        */
    int32_t *w_lr[NITRO_MAX_BLOCKS];                  /* learning-layer weights (updated)       */
    int32_t *w_head;                                  /* output layer [G][d_L] (if head)        */
} nitro_net_params;

/* Size in bytes of the network workspace: every block's state and output, and every weight
 * gradient. */
nitro_status nitro_net_query(const nitro_net_desc *net, size_t *workspace_bytes);

/* One training iteration (section 3.3): forward through every block, output layer and its
 * IntegerSGD update, then each block's local training and the IntegerSGD update of its learning
 * layer (gamma_inv) and forward layers (AF * gamma_inv). All gradients are taken at the weights
 * from before the iteration. Weights in `params` are updated in place.
 * Dropout (hp->dropout_conv_ppm, hp->dropout_lin_ppm > 0): each block's output is thinned after
 * its forward layers; a dropped element becomes 0, for the next block and the learning layer
 * alike, and passes no gradient back. The mask of block b: element i (flat NHWC / [n][d] order)
 * takes 64-bit word i mod 4 of Philox4x64-10 (Salmon et al., SC'11) at counter (i div 4 + 1, b,
 * dropout_step, 0) and key (dropout_seed, 0), and is dropped when the word's upper 32 bits are
 * below floor(p 2^32), p = ppm / 10^6. No rescaling of the kept elements (the next layer's
 * NITRO-Scaling sets the scale). The caller advances dropout_step between iterations.
 *   x       int8 input batch (NHWC, or [n][d] for an MLP);
 *   labels  int32 [n] in [0, G). */
nitro_status nitro_train_step(nitro_ctx *ctx, const nitro_net_desc *net,
                              const nitro_net_params *params, void *workspace,
                              const int8_t *x, const int32_t *labels, const nitro_hparams *hp);

/* Inference with the current weights (the accuracy protocol of section 4): the forward pass
 * through every block (section 3.2), then the network's prediction yhat = floor(f W^T / 2^8 d)
 * of the output layer on the last block's output f, or, without an output layer, of the last
 * block's learning layer on its input, and the predicted class: the first maximum of each row.
 *   workspace  laid out by nitro_net_query (a training workspace serves);
 *   x          int8 input batch;  yhat  int32 [n][G];  pred  int32 [n].
 * Labels are not needed; every block's n_classes must still be G > 0 (the shapes of the
 * training network). Weights are not changed. */
nitro_status nitro_net_infer(nitro_ctx *ctx, const nitro_net_desc *net,
                             const nitro_net_params *params, void *workspace, const int8_t *x,
                             int32_t *yhat, int32_t *pred);

/* nitro_train_step replayed from a HIP graph. The context keeps up to 16 captured iterations,
 * one per distinct key (compared by value: descriptors, parameter pointers, workspace, x,
 * labels, hyper-parameters, the context's stream and settings, the timing switch). A call whose
 * key has no graph captures one iteration on the context's stream and instantiates it (beyond
 * 16, in place of the least recently replayed, after synchronising the stream); every call then
 * launches its key's graph. A graph reads x and labels from the buffers it was captured with:
 * a caller changes the batch by writing into those buffers, or by passing other resident
 * buffers, which get graphs of their own (all of them share the one workspace, so replays run
 * in stream order). The context's stream must not be the legacy default stream (EINVAL).
 * Capture errors return the error of the failing call or NITRO_EHIP. nitro_kernel_timing and
 * nitro_destroy release every graph (synchronising the stream first). */
nitro_status nitro_train_step_graph(nitro_ctx *ctx, const nitro_net_desc *net,
                                    const nitro_net_params *params, void *workspace,
                                    const int8_t *x, const int32_t *labels, const nitro_hparams *hp);

/* The graph nitro_train_step_graph would replay for these arguments, captured and instantiated
 * now if the context has none for their key, and not launched: nothing runs on the GPU and no
 * weight changes. A training loop over several resident batches prepares each one's graph before
 * its first iteration, so that no capture happens between replays. Same arguments, limits and
 * errors as nitro_train_step_graph (preparing a 17th key replaces the least recently used). */
nitro_status nitro_train_step_graph_prepare(nitro_ctx *ctx, const nitro_net_desc *net,
                                            const nitro_net_params *params, void *workspace,
                                            const int8_t *x, const int32_t *labels,
                                            const nitro_hparams *hp);

/* Device pointer, inside a workspace laid out by nitro_net_query, of block b's output a_b
 * (int8), so that callers can inspect the forward activations after nitro_train_step. */
nitro_status nitro_net_block_output(const nitro_net_desc *net, void *workspace, int32_t b,
                                    int8_t **a_out);

/* Device pointers, inside a workspace laid out by nitro_net_query, of what a training iteration
 * leaves there for block b (for inspection; valid after the iteration's work has run):
 *   a_out    int8 block output (pooled if the block pools), NHWC or [n][d];
 *   act[j]   int8 output of forward layer j < n_layers - 1 (NULL for the last layer);
 *   code[j]  NITRO-ReLU region codes of layer j, as described at nitro_block_saved;
 *   yhat, e  int32 [n][G] learning-layer prediction and loss gradient;
 *   dw[j]    int64 weight gradient of forward layer j (KRSC / [out][in]);
 *   dw_lr    int64 [G][d] learning-layer weight gradient.
 * Unused entries are NULL. */
typedef struct {
    int8_t *a_out;
    int8_t *act[NITRO_MAX_LAYERS];
    uint8_t *code[NITRO_MAX_LAYERS];
    int32_t *yhat, *e;
    int64_t *dw[NITRO_MAX_LAYERS];
    int64_t *dw_lr;
} nitro_block_view;
nitro_status nitro_net_block_view(const nitro_net_desc *net, void *workspace, int32_t b,
                                  nitro_block_view *out);
/* The output layer's int32 [n][G] prediction and loss gradient and its int64 [G][d] weight
 * gradient inside the workspace (EINVAL when the network has no output layer). */
nitro_status nitro_net_head_view(const nitro_net_desc *net, void *workspace, int32_t **yhat,
                                 int32_t **e, int64_t **dw);

/* ------------------------------------------------------------------------------------------ */
/* Host-side helpers (no device work)                                                         */
/* ------------------------------------------------------------------------------------------ */

/* The division the kernels use (multiply by a precomputed reciprocal of the invariant
 * divisor), evaluated on the host: n / d with d >= 1 and |n| < 2^62, rounded per `round`. */
int64_t nitro_host_div(int64_t n, int64_t d, int32_t round);
/* NITRO-ReLU mean for alpha_inv (section 3.2.2) under `round`. */
int32_t nitro_host_relu_mu(int32_t alpha_inv, int32_t round);
/* Bound b of the integer Kaiming initialisation (section 3.3.1): weights are drawn uniformly from
 * [-b, b] with b = floor(128 * 1732 / (isqrt(fan_in) * 1000)), isqrt the integer square root.
 * Returns 0 for fan_in < 1. */
int32_t nitro_host_kaiming_bound(int64_t fan_in);

/* Per-kernel timing for profiling. enable = 1 (device timestamps): while enabled, every launch of a
 * timed kernel class records,
 * on the device, the wall-clock time from its first workgroup's start to its last workgroup's
 * end (this also works inside a graph replayed by nitro_train_step_graph). Classes: 0 the tiled
 * int8 MFMA conv forward kernel, 1 the tiled conv input-gradient kernel, 2 the conv
 * weight-gradient kernel over padded pixel planes (layers that take other kernels are not
 * timed). Enabling allocates the context's timing buffer once (ENOMEM) and restarts the count.
 * nitro_kernel_time synchronises the context's stream and returns the summed milliseconds and
 * the number of launches: of the launches enqueued since the last read or enable, or, when a
 * graph was captured with timing on, of the last replay. */
/* enable = 2 (events): every eager launch of a timed class (not one being captured into a graph)
 * is bracketed by two HIP events recorded on the stream it is launched on; nitro_kernel_time
 * then returns the summed event-to-event times of the launches since the last read (at most
 * 1024 per class). 0 disables timing. EINVAL for other values. */
nitro_status nitro_kernel_timing(nitro_ctx *ctx, int32_t enable);
nitro_status nitro_kernel_time(nitro_ctx *ctx, int32_t cls, double *ms, int64_t *launches);

/* Rate probe of the int8 matrix cores, which states the dense peak that the conv kernels'
 * throughput is priced against. One launch runs 8 independent v_mfma_i32_16x16x64_i8 chains per
 * wave on operands held in registers (no memory traffic but one 4-byte store per thread at the
 * end), with waves_per_simd (1..4) waves on every SIMD of every compute unit and iters (>= 1)
 * MFMAs per chain, timed with HIP events on the context's stream after a short warm-up launch.
 * *tops receives the rate achieved in 10^12 int8 ops per second (2 * 16 * 16 * 64 ops per MFMA).
 * Synchronous. Allocates and frees a result buffer of 1 KiB per workgroup (ENOMEM); EINVAL for a
 * null argument or a count out of range, EHIP for a failed launch or event. */
nitro_status nitro_mfma_rate(nitro_ctx *ctx, int32_t waves_per_simd, int32_t iters, double *tops);

#ifdef __cplusplus
}
#endif
#endif /* NITRO_H */
