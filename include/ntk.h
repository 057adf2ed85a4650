/*
 * ntk.h -- C ABI of the MI355X (gfx950) structured-derivatives empirical NTK library.
 *
 * The library computes the finite-width empirical neural tangent kernel
 *
 *     Theta(x1, x2) = [df(x1)/dtheta] [df(x2)/dtheta]^T            (O x O per input pair)
 *
 * (Section 3.1.1, Eq. ntk_def_main) for fully-connected and 3x3-convolutional
 * networks, without ever forming the Jacobian.  It follows the "structured
 * derivatives" method of Section 3.4: for every weight tensor theta^l it
 * contracts the smallest Jacobian sub-array of dy/dtheta^l (the layer input,
 * or its 3x3 patches for a convolution) with the primitive-output cotangents
 * df/dy of both batches, and sums the summands over layers (Eq.
 * expanded_ntk_main, Eq. mixed_product_example; per-layer formulas of
 * Section 4.1 for the FCN and the appendix "CNN NTK Complexity" for the CNN).
 *
 * The contractions run on the GPU in fp32 with fp32 accumulation (the paper's
 * experiments use 32-bit precision, appendix "Experimental Details").  The forward
 * pre-activations are accumulated in fp64 from the fp32 layer inputs and weights, so that
 * the activation's decisions (the ReLU sign) are those of the exact pre-activation; every
 * stored array (layer inputs, derivatives, cotangents, Theta) is fp32.
 *
 * Networks (the descriptor below):
 *   * FCN: n >= 1 DENSE layers.  Layer l maps d_l -> d_{l+1}:
 *       z_l = h_l W_l^T (+ b_l),  h_{l+1} = act_l(z_l),  h_0 = x,  f = z_last.
 *     The last layer must have act NONE (f is the last pre-activation).
 *   * CNN: 1..64 spatial layers, then one GAP layer (mean over the pixels), then
 *     one DENSE readout layer with act NONE and no bias.  The spatial layers, in any
 *     order, at least one of them with parameters:
 *       CONV3X3_SAME   z = 3x3 cross-correlation, stride 1, zero padding 1, weights
 *                      [Cout,3,3,Cin] (OHWI), optional bias [Cout];
 *       CONV1X1        pointwise: a dense layer at every pixel, weights [Cout,Cin],
 *                      optional bias [Cout];
 *       DWCONV3X3_SAME depthwise: channel c convolved with its own 3x3 filter, weights
 *                      [3,3,C], optional bias [C]; in == out;
 *       SCALE          z = h * w[c], weights [C], optional bias [C]; in == out;
 *       AVGPOOL2       mean over non-overlapping 2x2 windows (stride 2), no parameters,
 *                      act NONE; the image height and width must be even there.
 *     Activations are NHWC.  The three parametrised kinds take any activation.
 *     How each kind's weight-space Jacobian is structured, and how it is contracted:
 *     the 3x3 convolution is constant-block-diagonal (the outside-in or inside-out
 *     orders of NTK_OPT_CONV_ORDER), the pointwise one too (outside-in: Cout*Cin columns); the depthwise convolution is block-diagonal over
 *     channels and the scale layer block-diagonal over channels and output
 *     block-tiled over pixels (appendix "Block Diagonal", "Output Block-tiled"): their
 *     weight-space cotangents are per-channel pixel sums, 9*C and C columns; every
 *     bias is output block-tiled, its cotangent the pixel sum of the output cotangent
 *     (C columns).  These columns are contracted by the same split-K product as the
 *     outside-in 3x3 convolution columns.
 *
 * Conventions: act'(0) = 0 for ReLU; erf'(z) = 2/sqrt(pi) exp(-z^2).
 *
 * Ownership and streams: the caller owns every pointer it passes (parameters,
 * inputs, output); the library owns only its workspace, allocated by
 * ntk_init and released by ntk_free.  Work is enqueued on the handle's HIP
 * stream and returns before it finishes; the caller synchronises.  A handle
 * must not be used by two host threads at once, and two calls on the same
 * handle must be ordered on one stream (they share the workspace).
 *
 * Errors: every entry point returns NTK_OK (0) or a negative NTK_E_* code and,
 * when a handle exists, records a message readable with ntk_last_error.  No
 * C++ exception crosses this interface.  On NTK_E_ARG / NTK_E_SHAPE /
 * NTK_E_UNSUPPORTED nothing is enqueued and the output is left untouched.
 */
#ifndef NTK_H_
#define NTK_H_

#ifdef __cplusplus
extern "C" {
#endif

/* ---- return codes ---------------------------------------------------------------- */
#define NTK_OK             0
#define NTK_E_ARG         -1  /* null pointer, n <= 0, n > max, bad option value            */
#define NTK_E_SHAPE       -2  /* inconsistent model descriptor (dims do not chain, ...)      */
#define NTK_E_UNSUPPORTED -3  /* layer kind / activation / layer order not supported          */
#define NTK_E_OOM         -4  /* workspace allocation failed                                  */
#define NTK_E_HIP         -5  /* a HIP runtime call or kernel launch failed (message has it)  */

/* ---- layer kinds and activations ------------------------------------------------- */
#define NTK_DENSE          0
#define NTK_CONV3X3_SAME   1
#define NTK_GAP            2
#define NTK_DWCONV3X3_SAME 3
#define NTK_SCALE          4
#define NTK_AVGPOOL2       5
#define NTK_CONV1X1        6

#define NTK_ACT_NONE       0
#define NTK_ACT_RELU       1
#define NTK_ACT_ERF        2

typedef struct ntk_layer_desc {
    int kind;      /* NTK_DENSE, NTK_CONV3X3_SAME, NTK_CONV1X1, NTK_DWCONV3X3_SAME,
                      NTK_SCALE, NTK_AVGPOOL2 or NTK_GAP                                  */
    int in;        /* input features / input channels (ignored for AVGPOOL2 and GAP)      */
    int out;       /* output features / output channels (ignored for AVGPOOL2 and GAP)    */
    int act;       /* activation applied to this layer's output (NTK_ACT_*; AVGPOOL2 and
                      GAP: NONE)                                                          */
    int has_bias;  /* 1 if the layer has a bias vector of length `out` (not AVGPOOL2, GAP,
                      or the CNN readout)                                                 */
} ntk_layer_desc;

typedef struct ntk_model_desc {
    int n_layers;                  /* number of entries in `layers`                      */
    const ntk_layer_desc* layers;  /* copied by ntk_init; need not outlive the call      */
    int in_h, in_w, in_c;          /* input shape: FCN uses in_h = in_w = 1, in_c = d_0  */
    int out_dim;                   /* O, the number of network outputs                   */
} ntk_model_desc;

typedef struct ntk_handle ntk_handle;

/* ---- options (ntk_set_option) ---------------------------------------------------- */
/* NTK_OPT_SYMMETRIC: 1 (default) = when X2 == X1 and n2 == n1, run the forward and
 * backward passes once and compute only the upper triangle of output tiles,
 * mirroring the transposed O x O blocks (Theta(x,x')[o1,o2] = Theta(x',x)[o2,o1]);
 * 0 = always treat X1 and X2 as two batches.                                          */
#define NTK_OPT_SYMMETRIC   1
/* NTK_OPT_CONV_ORDER: contraction order of the convolutional summands (appendix
 * "No Structure": outside-in vs inside-out; appendix "CNN NTK Complexity").
 * 0 = auto (per layer, the faster order by the paper's CNN cost model, the inside-out
 *     FLOPs weighted by the measured time per FLOP of the pair-sum kernels on MI355X
 *     relative to the matrix-core path: 9 for images of at most 16 pixels, 40 above),
 * 1 = outside-in (per-sample weight-space Jacobian, then J1 J2^T),
 * 2 = inside-out (patch-pair Gram times cotangent Gram, summed over pixel pairs).  */
#define NTK_OPT_CONV_ORDER  2
#define NTK_CONV_ORDER_AUTO        0
#define NTK_CONV_ORDER_OUTSIDE_IN  1
#define NTK_CONV_ORDER_INSIDE_OUT  2
/* NTK_OPT_OUTPUT: which part of the O x O block of every input pair is computed (the
 * pseudo-NTK of the appendix "Pseudo-NTK"; compute-wise these have O = 1):
 *   NTK_OUTPUT_FULL  (default) the whole block Theta(x1, x2)[o1, o2];
 *   NTK_OUTPUT_TRACE its trace sum_o Theta(x1, x2)[o, o] (divide by O for the mean of the
 *                    O diagonal blocks);
 *   NTK_OUTPUT_LOGIT Theta(x1, x2)[o*, o*] for the logit o* set by NTK_OPT_LOGIT (the NTK of
 *                    that one output; the backward pass runs for it alone).
 * NTK_OPT_LOGIT: o*, 0 <= o* < O (default 0).
 * NTK_OPT_BATCH: which input pairs are computed:
 *   NTK_BATCH_FULL     (default) every pair (n1, n2);
 *   NTK_BATCH_DIAGONAL only the pairs (n, n), Theta(x1_n, x2_n); needs n1 == n2.
 * The layout of theta follows (row-major, fp32):
 *   FULL  x FULL      [n1, n2, O, O]      FULL  x DIAGONAL  [n, O, O]
 *   TRACE/LOGIT x FULL [n1, n2]           TRACE/LOGIT x DIAGONAL [n]                      */
#define NTK_OPT_OUTPUT      3
#define NTK_OUTPUT_FULL     0
#define NTK_OUTPUT_TRACE    1
#define NTK_OUTPUT_LOGIT    2
#define NTK_OPT_LOGIT       4
#define NTK_OPT_BATCH       5
#define NTK_BATCH_FULL      0
#define NTK_BATCH_DIAGONAL  1
/* NTK_OPT_METHOD: how Theta is computed.
 *   NTK_METHOD_STRUCTURED (default) the structured-derivatives method of Section 3.4;
 *   NTK_METHOD_JACOBIAN   the Jacobian-contraction baseline of Section 3.2: the per-sample
 *                         Jacobian df/dtheta (reverse mode, O vector-Jacobian products) is
 *                         formed explicitly, block by block, and Theta = J(x1) J(x2)^T is
 *                         contracted on the matrix cores (N1 N2 O^2 P multiply-adds).  Conv
 *                         layers then use the outside-in order.  It exists for comparison;
 *                         the first call on a handle allocates its Jacobian buffers.
 * Every variant of NTK_OPT_OUTPUT / NTK_OPT_BATCH is available with both methods.          */
#define NTK_OPT_METHOD             6
#define NTK_METHOD_STRUCTURED      0
#define NTK_METHOD_JACOBIAN        1
/* NTK_OPT_GRAPH: 1 = ntk_compute records its launches into a HIP graph on the first call and
 * replays the graph on later calls with the same arguments (parameter, input and output
 * pointers, batch sizes, options) -- the contents of the buffers may change; other arguments
 * record a new graph.  Cuts the per-launch host overhead of small problems.  Not used while
 * per-kernel timing is enabled or when the caller's stream is itself being captured.
 * 0 (default) = launch eagerly.                                                           */
#define NTK_OPT_GRAPH              7

/*
 * ntk_init -- validate a model descriptor, plan and allocate the workspace.
 *   model       descriptor (copied).
 *   max_n1/2    largest batch sizes later passed to ntk_compute (> 0).
 *   hip_stream  hipStream_t the work is enqueued on; NULL = the default stream.
 *   out         receives the new handle; set to NULL on any error.
 * Returns NTK_OK, NTK_E_ARG, NTK_E_SHAPE, NTK_E_UNSUPPORTED, NTK_E_OOM or NTK_E_HIP.
 * Size limit: every array the kernels index -- theta [max_n1, max_n2, O, O], an input batch,
 * each layer's inputs and cotangents for max_n1 + max_n2 samples and all O outputs, the
 * weight-space cotangent columns of a CNN, the split-K partials -- must hold fewer than 2^31
 * elements (the kernels form rows and offsets as 32-bit ints).  A descriptor and batch sizes
 * that break this are refused with NTK_E_UNSUPPORTED, naming the array, before any HIP call
 * and before anything is allocated; larger problems are computed in blocks of samples
 * (Theta(X1[R1], X2[R2]) is the block [R1, R2] of Theta(X1, X2)).
 * The device is the one current on the calling thread; later calls must keep it current.
 */
int ntk_init(const ntk_model_desc* model, int max_n1, int max_n2, void* hip_stream,
             ntk_handle** out);

/*
 * ntk_compute -- enqueue Theta(X1, X2) on the handle's stream.
 *   params  host array of device pointers, one per parameter tensor in layer
 *           order, weight first then bias (if has_bias): dense weight [out, in]
 *           row-major, conv weight [Cout, 3, 3, Cin] (OHWI), pointwise weight
 *           [Cout, Cin], depthwise weight
 *           [3, 3, C], scale weight [C], every bias [out]; AVGPOOL2 and GAP have none.
 *   X1      device [n1, in_c] (FCN) or [n1, in_h, in_w, in_c] NHWC (CNN), fp32.
 *   X2      device, same layout with n2 rows.  X2 == X1 with n2 == n1 selects the
 *           symmetric schedule (see NTK_OPT_SYMMETRIC).
 *   theta   device [n1, n2, O, O] fp32 row-major:
 *           theta[((n1*N2 + n2)*O + o1)*O + o2] = Theta(x1_{n1}, x2_{n2})[o1, o2],
 *           or the smaller array that NTK_OPT_OUTPUT / NTK_OPT_BATCH select (see there).
 *           Every entry is written.  theta must not overlap the inputs.
 * NTK_E_ARG also when NTK_OPT_LOGIT is not below O, or NTK_BATCH_DIAGONAL with n1 != n2.
 * Stream-ordered and asynchronous.  Deterministic: two calls with the same inputs
 * give bit-identical theta (no atomics).
 */
int ntk_compute(ntk_handle* h, const float* const* params, const float* X1, int n1,
                const float* X2, int n2, float* theta);

/*
 * ntk_vector_product -- enqueue out = Theta(X1, X2) v without forming Theta (the NTK-vector
 * product of Section 3.3, Eq. ntk_vp_main): the VJP of batch 2 at v gives the weight-space
 * vector theta_c = J(X2)^T v, and the JVP of batch 1 along theta_c gives J(X1) theta_c.
 *   params, X1, n1, X2, n2  as for ntk_compute.
 *   v    device [n2, O] fp32: v[n2*O + o2].
 *   out  device [n1, O] fp32: out[n1*O + o1] = sum_{n2, o2} Theta(x1_{n1}, x2_{n2})[o1, o2] v[n2, o2].
 * Time about 3 forward passes of the batches (no N1 N2 O^2 term).  The output and batch
 * variants and NTK_OPT_METHOD do not apply.  Every layer kind is supported.  The first call on a handle allocates the
 * weight-space vector (one float per parameter) and the tangent buffers.  Stream-ordered,
 * asynchronous, deterministic; NTK_E_ARG for null pointers or sizes out of range.
 */
int ntk_vector_product(ntk_handle* h, const float* const* params, const float* X1, int n1,
                       const float* X2, int n2, const float* v, float* out);

/* ---- an entry point that allocates nothing ---------------------------------------
 * ntk_compute_static -- for callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  Enqueues the full theta
 * [n1, n2, O, O] on `hip_stream` (NULL = the default stream), as ntk_compute does with the
 * default options (structured method, full output, the symmetric schedule when X2 == X1 and
 * n2 == n1, automatic conv contraction order), but without a handle: the descriptor is
 * validated and planned on every call (host work only), and the workspace is one fixed device
 * array of NTK_STATIC_SCRATCH_BYTES inside the library per GPU, which stays resident until the
 * process ends.  The call allocates and frees no device memory, and creates no streams or
 * events.
 *   model, params, X1, n1, X2, n2, theta  as for ntk_init and ntk_compute.
 * Returns NTK_OK, NTK_E_ARG, NTK_E_SHAPE, NTK_E_UNSUPPORTED or NTK_E_HIP; the message is read
 * with ntk_last_error(NULL).  NTK_E_UNSUPPORTED, with nothing enqueued, also when the
 * workspace of this model and these batch sizes exceeds NTK_STATIC_SCRATCH_BYTES (the message
 * gives the bytes needed; use ntk_init then).
 * Every call on a GPU uses that GPU's one array and leaves its contents there (nothing in it
 * needs clearing between calls): calls that overlap on one GPU -- on different streams or
 * from different host threads -- race, and the caller must order them.  The first call with a
 * device current looks up the array's device address.
 */
#define NTK_STATIC_SCRATCH_BYTES (64 * 1024 * 1024)
int ntk_compute_static(const ntk_model_desc* model, const float* const* params, const float* X1, int n1,
                       const float* X2, int n2, float* theta, void* hip_stream);

/* ntk_free -- release the workspace and the handle.  NULL is a no-op.  Synchronises
 * the handle's stream first. */
int ntk_free(ntk_handle* h);

/* ntk_last_error -- message of the last failed call on `h` ("" if none).  With
 * h == NULL, the message of the last failed ntk_init on this thread. */
const char* ntk_last_error(const ntk_handle* h);

/* ntk_set_option -- set NTK_OPT_* (see above).  NTK_E_ARG for an unknown option/value. */
int ntk_set_option(ntk_handle* h, int option, int value);

/* ntk_set_stream -- change the stream later work is enqueued on (NULL = default). */
int ntk_set_stream(ntk_handle* h, void* hip_stream);

/* ntk_workspace_bytes -- bytes of device workspace the handle holds. */
long long ntk_workspace_bytes(const ntk_handle* h);

/* ---- per-kernel timing ------------------------------------------------------------
 * When enabled, every kernel launch of ntk_compute is bracketed by HIP events on the
 * handle's stream and the elapsed times are accumulated per kernel class.
 * ntk_profile_read synchronises the stream, writes up to `max` entries (class name,
 * total milliseconds, number of launches) and resets the accumulators.  It returns the
 * number of classes written (>= 0) or a negative error code.  Names stay valid for the
 * life of the handle. */
int ntk_profile_enable(ntk_handle* h, int enable);
int ntk_profile_read(ntk_handle* h, const char** names, double* total_ms,
                     long long* launches, int max);

/* ---- device diagnostics ----------------------------------------------------------
 * ntk_device_info -- number of compute units and peak engine clock (kHz) of the device
 * current on the calling thread.  NTK_E_ARG for a null pointer, NTK_E_HIP on a HIP error.
 *
 * ntk_mfma_peak -- measured matrix-core ceiling of the current device in TFLOP/s:
 * which = 0 for v_mfma_f32_32x32x2_f32 (fp32), 1 for v_mfma_f64_16x16x4_f64 (fp64).  A
 * kernel of independent MFMA chains (four 4-wave workgroups per compute unit) is timed
 * with HIP events on a private stream; the call is synchronous and allocates (then frees)
 * a small output buffer.  Returns NTK_OK, NTK_E_ARG, NTK_E_OOM or NTK_E_HIP. */
int ntk_device_info(int* num_cu, int* clock_khz);
int ntk_mfma_peak(int which, double* tflops);

#ifdef __cplusplus
}
#endif
#endif /* NTK_H_ */
