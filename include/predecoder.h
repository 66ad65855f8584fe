/*
 * predecoder.h -- C ABI of the MI355X (gfx950) pre-decoder hot path.
 *
 * Implements the inference step of the local 3D-convolutional pre-decoder for
 * the rotated surface code ("Fast and accurate AI-based pre-decoders for
 * surface codes", arXiv 2604.12841): a fully convolutional 3D CNN over the
 * space-time volume of detector events (Sec. IV.B, Fig. ConvArch), whose four
 * output channels are read as data-qubit Z/X corrections and X/Z
 * stabilizer-measurement (timelike) corrections (Sec. IV.B.6, Eqs.
 * ZcorreJK-SynZCorrJK), thresholded at logit > 0 (the sigmoid of the BCE
 * objective, Sec. IV.B.5), and applied to the syndrome history to give the
 * residual syndrome that is handed to a global decoder (Eqs. Resk1X, ReskG1X,
 * Resk1Z, ReskG1Z).
 *
 * Geometry.  Distance d (odd, >= 3), T rounds.  Stabilizers live on the
 * (d+1) x (d+1) plaquette grid, sites (i, j) with 0 <= i, j <= d:
 *   X site  <=>  (i + j) even and 1 <= i <= d-1
 *   Z site  <=>  (i + j) odd  and 1 <= j <= d-1
 * Plaquette (i, j) acts on the data qubits (i-1, j-1), (i-1, j), (i, j-1),
 * (i, j) that lie inside [0, d-1]^2 (weight 4 in the bulk, weight 2 on the
 * boundary).  X_L is a horizontal and Z_L a vertical string (Sec. III, Fig. SurfaceCodeExamp).
 * Data qubit (r, c) is identified with grid site (r, c), r, c < d.  There are
 * K = (d^2 - 1) / 2 stabilizers of each type (Eqs. DetectorX/DetectorZ).
 *
 * Bit-packed formats (all LSB-first: bit b of a sample row is bit (b & 63) of
 * 64-bit word (b >> 6); every sample row is a whole number of words; padding
 * bits are ignored on input and written as 0 on output):
 *   detectors / residual, W_det = predecoder_det_words(d, T) words per sample:
 *     b = t * (d^2 - 1) + n; n < K enumerates the X sites in row-major (i, j)
 *     order, n >= K the Z sites in row-major order.  A detector bit is the
 *     XOR of one stabilizer's outcomes in rounds t and t-1 (Sec. IV.B.1).
 *   flips, W_flip = predecoder_flip_words(d, T) words per sample:
 *     b = t * (3 d^2 - 1) + n with n running over
 *       [0, d^2)          Z data-qubit correction (output channel 0), (r, c) row-major
 *       [d^2, 2 d^2)      X data-qubit correction (output channel 1)
 *       [2 d^2, 2 d^2+K)  X-stabilizer measurement flip (channel 2), X-site order
 *       [2 d^2+K, 3d^2-1) Z-stabilizer measurement flip (channel 3), Z-site order
 *
 * Residual (Eqs. Resk1X..ReskG1Z, with a measurement flip in round t also
 * flipping round t+1, and nothing before round 0):
 *   R_X[t](s) = D_X[t](s) ^ m_X[t](s) ^ m_X[t-1](s) ^ XOR_{q in supp(s)} z_corr[t](q)
 *   R_Z[t](s) = D_Z[t](s) ^ m_Z[t](s) ^ m_Z[t-1](s) ^ XOR_{q in supp(s)} x_corr[t](q)
 * applied at every round 0 <= t < T (including the last one).
 *
 * Input layouts (pd_options.layout):
 *   PD_LAYOUT_PLAQUETTE (default): the (d+1) x (d+1) plaquette grid above,
 *     two channels (X-type, Z-type detector events at their stabilizer
 *     sites, zero elsewhere).
 *   PD_LAYOUT_PAPER: the paper's own encoding (Sec. IV.B.1, Fig. StabMap,
 *     Eqs. encTrainX1-encTrainX4): the D x D grid of data qubits (D = d), every
 *     stabilizer drawn onto one qubit of its support -- a weight-four X (Z)
 *     stabilizer onto its top-left (top-right) qubit, a weight-two X
 *     stabilizer (left / right edge) onto its upper qubit, a weight-two Z
 *     stabilizer (top / bottom edge) onto its right qubit -- and four
 *     channels: x_type, z_type (the detector events of the stabilizer drawn
 *     at the qubit), x_present, z_present (its weight / 4, i.e. 1 or 0.5).
 *     pd_options.first_round / last_round name the basis the logical qubit
 *     is prepared in before round 0 / measured in after round T-1: Z clears
 *     x_present in that round, X clears z_present, PD_BOUNDARY_NONE neither
 *     (a block in the middle of a stream).  The output channels are read at
 *     the same positions: channels 0/1 at every qubit, channel 2 (3) at the
 *     qubit an X (Z) stabilizer is drawn onto.  Logits are [4][T][d][d].
 *
 * Network.  A list of conv3d layers (stride 1, no dilation, zero padding
 * (k-1)/2, cross-correlation as in PyTorch Conv3d):
 *   layers[0].c_in == 2 (plaquette layout) or 4 (paper layout)
 *   layers[l].c_in == layers[l-1].c_out
 *   layers[n-1]: the output layer, c_out == 4, act == PD_ACT_NONE: a 1x1x1
 *                head, or (paper layout) a 3x3x3 layer as in Table models.
 * Hidden layers apply their activation; GELU is the tanh form
 * 0.5 y (1 + tanh(sqrt(2/pi) (y + 0.044715 y^3))) (Table hyperparameters).
 * Weights are host fp32, layer after layer, each as w[c_out][c_in][kt][ki][kj]
 * followed by b[c_out]; tap (kt, ki, kj) multiplies x[t+kt-p][i+ki-p][j+kj-p].
 *
 * Precision.  PD_DTYPE_BF16: weights and every conv/head input are rounded
 * to bf16 (round to nearest even), products are accumulated in fp32, biases
 * and the activation are fp32, logits are fp32.  PD_DTYPE_FP32: fp32 end to
 * end.  flip = (logit > 0); a logit of exactly 0 is no flip.  Results are
 * bit-reproducible for a given handle and batch size; small batches split the
 * conv K loops over several workgroups, so two batch sizes can differ in the
 * fp32 summation order, and through an activation rounded to the other bf16
 * neighbour, by up to a few 1e-3 in the logits.
 * PD_DTYPE_FP8 (the paper deploys its models in FP8, Sec. VI, without
 * stating the scaling; this is the library's reading): OCP E4M3 values (4
 * exponent bits, bias 7, 3 mantissa bits, largest finite 448).  Each output
 * channel of each layer gets a power-of-two weight scale 2^e, e the smallest
 * integer with max |w| / 2^e <= 448 over the channel's weights, and its
 * weights are used as e4m3(w / 2^e) * 2^e; every conv or head input is an
 * E4M3 value with no scale (the input planes, 0, 1/2 and 1, are exact);
 * rounding is to nearest, ties to even, magnitudes above 448 saturate.
 * Products are accumulated in fp32; bias, activation and logits are fp32.
 * Same reproducibility rule as bf16; an activation rounded to the other
 * E4M3 neighbour moves the logits further (the parity tolerance is larger).
 *
 * Supported shapes (others give PD_ERR_UNSUPPORTED): 3 <= d <= 63,
 * 1 <= T <= 1023; hidden layers k == 3; output layer k == 1, or k == 3 on
 * the paper layout.  BF16 and FP8: hidden widths 64, 128 or 256 (a layer
 * after a 256-wide one needs a 3x3x3 output layer); FP8 needs two hidden
 * layers when the output layer is 1x1x1.  FP32 (plaquette layout only):
 * hidden widths 8 .. 128, multiples of 8.  5x5x5 networks (Model 3 of
 * Table models): the paper layout, PD_DTYPE_BF16, every layer k == 5 (the
 * output layer too), at least two hidden layers, all of one width, 64 or
 * 128.
 *
 * Errors.  Every function is nothrow and never aborts.  Host-checkable misuse
 * gives PD_ERR_INVALID_ARG before any device call; a failed HIP call or
 * launch (including "no device") gives PD_ERR_DEVICE; a failed allocation
 * gives PD_ERR_OUT_OF_MEMORY.  After an error the outputs are unspecified
 * and the handle stays usable.
 *
 * Ownership and streams.  Input/output buffers of run/residual/unpack are
 * caller-owned DEVICE memory.  The handle owns its copy of the weights, its
 * workspace and its tables.  Work is enqueued on the caller's HIP stream
 * (hipStream_t passed as void*; NULL = the null stream) and the host never
 * waits for it, except in predecoder_stage_times.  One handle must not be
 * used from two streams at once (the workspace is shared): use one handle
 * per stream.
 */
#ifndef PREDECODER_H
#define PREDECODER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum pd_status {
  PD_OK = 0,
  PD_ERR_INVALID_ARG = 1,
  PD_ERR_UNSUPPORTED = 2,
  PD_ERR_OUT_OF_MEMORY = 3,
  PD_ERR_DEVICE = 4,
  PD_ERR_TOO_LARGE = 5 /* predecoder_run_static: the batch needs more than its static array */
} pd_status;

typedef enum pd_act { PD_ACT_NONE = 0, PD_ACT_GELU_TANH = 1, PD_ACT_RELU = 2 } pd_act;

typedef enum pd_dtype { PD_DTYPE_FP32 = 0, PD_DTYPE_BF16 = 1, PD_DTYPE_FP8 = 2 } pd_dtype;

typedef enum pd_layout { PD_LAYOUT_PLAQUETTE = 0, PD_LAYOUT_PAPER = 1 } pd_layout;

/* Basis of the logical preparation / final measurement next to a block. */
typedef enum pd_boundary { PD_BOUNDARY_NONE = 0, PD_BOUNDARY_Z = 1, PD_BOUNDARY_X = 2 } pd_boundary;

/* Options of predecoder_create_ex (see "Input layouts" above).  first_round
 * and last_round must be PD_BOUNDARY_NONE on the plaquette layout. */
typedef struct pd_options {
  int32_t layout;      /* pd_layout */
  int32_t first_round; /* pd_boundary: basis prepared before round 0 */
  int32_t last_round;  /* pd_boundary: basis measured after round T-1 */
} pd_options;

/* One conv3d layer: k x k x k kernel, c_in -> c_out, activation act. */
typedef struct pd_layer {
  int32_t c_in;
  int32_t c_out;
  int32_t k;
  int32_t act;
} pd_layer;

typedef struct pd_predecoder pd_predecoder; /* opaque */

/* Builds a pre-decoder for distance d and T rounds (Sec. IV.B; the network
 * is fully convolutional, so the same weights apply to any (d, T)).
 * weights: host fp32, n_weights == predecoder_weight_count(layers, n_layers),
 *          copied (the caller keeps ownership).
 * dtype:   PD_DTYPE_BF16, PD_DTYPE_FP8 or PD_DTYPE_FP32.
 * max_batch: largest batch any later call may pass; sizes the workspace.
 * out:     receives the handle (NULL on error).
 * Allocates device memory on the current HIP device; launches nothing. */
pd_status predecoder_create(const float* weights, size_t n_weights, int32_t d, int32_t T,
                            const pd_layer* layers, int32_t n_layers, int32_t dtype,
                            int32_t max_batch, pd_predecoder** out);

/* predecoder_create with options (opts NULL = plaquette layout, no boundary
 * rounds): the input layout of Sec. IV.B.1 and the bases of the preparation
 * and final measurement.  Invalid option values give PD_ERR_INVALID_ARG; the
 * paper layout with PD_DTYPE_FP32 gives PD_ERR_UNSUPPORTED. */
pd_status predecoder_create_ex(const float* weights, size_t n_weights, int32_t d, int32_t T,
                               const pd_layer* layers, int32_t n_layers, int32_t dtype,
                               int32_t max_batch, const pd_options* opts, pd_predecoder** out);

/* The whole hot path for `batch` independent volumes (Sec. IV.B.6):
 * unpack -> conv layers (+bias, activation) -> head -> threshold ->
 * residual and bit repack.
 * det:      device, [batch][W_det] uint64, packed detectors (read only).
 * flips:    device, [batch][W_flip] uint64, packed thresholded corrections.
 * residual: device, [batch][W_det] uint64, packed residual syndrome.
 * logits:   device or NULL; if given, [batch][4][T][H][H] fp32 outputs of
 *           the last layer at every grid site (channel order as in `flips`;
 *           H = d + 1 on the plaquette layout, d on the paper layout).
 * 1 <= batch <= max_batch.  Asynchronous on hip_stream.  The run works in the
 * handle's workspace (activations, parked sums, the hidden kernel's unit
 * counters): runs of one handle must not overlap (one stream, or the caller
 * orders them); separate handles are independent. */
pd_status predecoder_run(pd_predecoder* h, void* hip_stream, const uint64_t* det, int32_t batch,
                         uint64_t* flips, uint64_t* residual, float* logits);

/* The residual stage alone (Eqs. Resk1X..ReskG1Z) from caller-given packed
 * flips: det [batch][W_det], flips [batch][W_flip] -> residual [batch][W_det],
 * all device.  Asynchronous on hip_stream. */
pd_status predecoder_residual(pd_predecoder* h, void* hip_stream, const uint64_t* det,
                              const uint64_t* flips, int32_t batch, uint64_t* residual);

/* The unpack stage alone (Sec. IV.B.1, Eqs. encTrainX1-4: the input planes
 * of the handle's layout): det [batch][W_det] -> planes, device,
 * [batch][T][H][H][c_in] (c_in = 2 on the plaquette layout, 4 on the paper
 * layout) as bf16 bit patterns (uint16) for PD_DTYPE_BF16 and
 * PD_DTYPE_FP8, fp32 for PD_DTYPE_FP32.
 * Asynchronous on hip_stream. */
pd_status predecoder_unpack(pd_predecoder* h, void* hip_stream, const uint64_t* det,
                            int32_t batch, void* planes);

/* The path up to hidden layer `layer` (0-based, a layer before the output
 * layer or head): its output activations as the next layer reads them --
 * after bias, activation and rounding to the handle's precision -- copied to
 * out, device, [batch][T][H][H][c_out] (bf16 bit patterns as uint16 for
 * PD_DTYPE_BF16, E4M3 codes as uint8 for PD_DTYPE_FP8).  For inspecting and
 * testing one layer at a time (Sec. IV.B, Fig. ConvArch: the activations
 * between the conv layers); a head that predecoder_run fuses into that layer
 * is not run.  On a residual network (predecoder_create_resnet) `layer`
 * counts its convs block by block -- conv1, the 1x1x1 projection if the
 * block has one, conv2 (with the shortcut added and the activation applied)
 * -- up to but not including the last block's conv2 (the output layer), and
 * c_out is that conv's width (Fig. Model8Representation).
 * PD_ERR_INVALID_ARG for a layer out of range, PD_ERR_UNSUPPORTED for
 * PD_DTYPE_FP32 and for the projection of an fp8 residual network (it is
 * computed inside the next conv, never stored).  Asynchronous on
 * hip_stream. */
pd_status predecoder_activations(pd_predecoder* h, void* hip_stream, const uint64_t* det,
                                 int32_t batch, int32_t layer, void* out);

/* Number of timed stages of predecoder_run: unpack, one per layer (the last
 * one is the head with its threshold), and the residual/repack stage. */
int32_t predecoder_num_stages(const pd_predecoder* h);

/* Runs the full path n_iter times on hip_stream with HIP events between the
 * stages and writes the mean milliseconds of each stage to ms_per_stage
 * (host, predecoder_num_stages(h) floats).  Arguments as predecoder_run
 * (logits not written).  Blocks the host until the stream has drained. */
pd_status predecoder_stage_times(pd_predecoder* h, void* hip_stream, const uint64_t* det,
                                 int32_t batch, uint64_t* flips, uint64_t* residual, int32_t n_iter,
                                 float* ms_per_stage);

/* Frees every device allocation of the handle.  NULL is ignored. */
void predecoder_destroy(pd_predecoder* h);

/* Static, human-readable name of a status code. */
const char* predecoder_status_string(pd_status s);

/* ceil(T (d^2 - 1) / 64): detector/residual words per sample; -1 on bad args. */
int64_t predecoder_det_words(int32_t d, int32_t T);

/* ceil(T (3 d^2 - 1) / 64): flip words per sample; -1 on bad args. */
int64_t predecoder_flip_words(int32_t d, int32_t T);

/* Sum over layers of c_out * c_in * k^3 + c_out (weights plus biases, the
 * parameter count of Table models); 0 on bad args. */
size_t predecoder_weight_count(const pd_layer* layers, int32_t n_layers);

/* ---- Recorded runs (HIP graphs) ----
 *
 * predecoder_graph_create records one predecoder_run of `batch` samples with
 * these buffers (device pointers, as for predecoder_run) into a HIP graph;
 * predecoder_graph_launch replays it on hip_stream, reading whatever det then
 * holds and writing flips / residual / logits (the same work and results as
 * predecoder_run, with one launch on the host).  Creating runs the path once
 * eagerly (on a stream of the graph's own, synchronously) so that the
 * handle's buffers are in the state every run starts from.  The graph uses
 * the handle's workspace: replays and runs of the same handle must not
 * overlap.  For latency-bound small batches (the paper times its models with
 * graph replays, Sec. VI). */
typedef struct pd_graph pd_graph; /* opaque */
pd_status predecoder_graph_create(pd_predecoder* h, const uint64_t* det, int32_t batch, uint64_t* flips,
                                  uint64_t* residual, float* logits, pd_graph** out);
pd_status predecoder_graph_launch(pd_graph* g, void* hip_stream);
void predecoder_graph_destroy(pd_graph* g); /* NULL is a no-op; waits for the device */

/* ---- A run that allocates nothing ----
 *
 * For callers that cannot allocate device memory while they run the path:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation.  predecoder_run_static takes the arguments of predecoder_run
 * and runs the same kernels, but keeps the workspace -- input planes,
 * activation buffers, projection outputs of residual networks, flip nibbles
 * and the parked sums of split K loops -- in a static device array of
 * PD_STATIC_SCRATCH_BYTES bytes that the library holds on every device it
 * runs on until the process ends, instead of the handle's own workspace.  It
 * calls no allocating routine (the handle is made beforehand with
 * predecoder_create*, which does allocate).
 *   Size: with S = (T + 2)(H + 2)^2 padded voxels and V = T H^2 voxels per
 *   sample, each region rounded up to 256 bytes: batch S c_in e (planes; e = 4
 *   for PD_DTYPE_FP32, else 2), two (residual networks: three) activation
 *   buffers of batch S cmax a (cmax the widest activation row; a = 4 fp32, 2
 *   bf16, 1 fp8), for residual networks batch S pmax 2 (the widest projection),
 *   and batch V (flip nibbles) must fit, else PD_ERR_TOO_LARGE before any
 *   device work.  What is left holds the parked sums of small batches' split K
 *   loops (128 KiB per unit, up to the handle's one per compute unit); with
 *   fewer units a layer may split less than predecoder_run splits it, and the
 *   results then differ by the fp32 summation order, as two batch sizes can.
 *   With room for all units the results are bit-identical to predecoder_run's.
 *   (Batch 1 with 128 channels on the plaquette grid needs about 2 MB before
 *   the parked sums at d = 13 and 20 MB at d = 31.)
 * Every call on one device uses that device's one array, which keeps the last
 * call's contents: each call clears what must start at zero (with a fill
 * kernel on hip_stream, no memset), and calls that overlap on one device --
 * from two streams or threads, with any handles -- race and give wrong
 * results; the caller serialises them.  Asynchronous on hip_stream; the first
 * call on a device looks up the array's device address (no allocation). */
#define PD_STATIC_SCRATCH_BYTES (64u << 20)
pd_status predecoder_run_static(pd_predecoder* h, void* hip_stream, const uint64_t* det, int32_t batch,
                                uint64_t* flips, uint64_t* residual, float* logits);

/* ---- Residual networks (Model 6, Sec. VI, Fig. Model8Representation) ----
 *
 * A block {c_in, c_mid, c_out, act}: conv1 (3x3x3, c_in -> c_mid) and
 * BatchNorm, the activation, conv2 (3x3x3, c_mid -> c_out) and BatchNorm, plus
 * the shortcut -- the block's input when c_in == c_out, else a 1x1x1
 * projection with bias -- then the activation, except after the last block,
 * whose c_out = 4 channels are the logits.  BatchNorm is the inference form
 * (x - running mean) / sqrt(running var + 1e-5) * scale + shift.  Model 6 is
 * {4,512,512}, {512,512,512} x 2, {512,512,4} with GELU (42,593,296 trainable
 * parameters; the running statistics add 2 floats per BatchNorm channel).
 * Weights, per block: conv1 w[c_mid][c_in][3][3][3], b[c_mid]; BatchNorm1
 * scale, shift, running mean, running variance [c_mid] each; conv2
 * w[c_out][c_mid][3][3][3], b[c_out]; BatchNorm2 (four [c_out]); projection
 * w[c_out][c_in], b[c_out] when c_in != c_out.
 * Precision: BatchNorm is folded into its conv at create (g = scale /
 * sqrt(var + eps) in fp64; weights bf16(fp32(w g)); bias fp32((b - mean) g +
 * shift)); projection weights bf16; every tensor stored between kernels
 * (activations, projection outputs) bf16; the conv2 sum plus the shortcut is
 * taken in fp32 before the activation.  PD_DTYPE_FP8: the folded weights
 * fp32(w g) and the projection weights as E4M3 codes with one power-of-two
 * scale per output channel (the fp8 reading of the plain networks), every
 * stored tensor E4M3.  The projections are computed inside the convs that
 * use them: the first block's (from its 2 or 4 input channels) in conv2's
 * epilogue, the last block's (when its c_in == c_mid) in the output conv;
 * fp8 handles allow no other projection.  Supported: PD_DTYPE_BF16 and
 * PD_DTYPE_FP8, c_mid in {64, 128, 256, 512}, c_out == c_mid inside the
 * network (others PD_ERR_UNSUPPORTED).  predecoder_run / residual / unpack / stage_times /
 * destroy take the handle like any other (stages: unpack, one per block,
 * residual); predecoder_activations returns the output of any conv but the
 * last (see there). */
typedef struct pd_block {
  int32_t c_in, c_mid, c_out; /* conv1: c_in -> c_mid, conv2: c_mid -> c_out */
  int32_t act;                /* pd_act after conv1 and after the shortcut add */
} pd_block;

/* Floats of a residual network's weights (layout above); 0 for invalid blocks. */
size_t predecoder_resnet_weight_count(const pd_block* blocks, int32_t n_blocks);

/* predecoder_create_ex for a residual network: blocks[0].c_in = 2
 * (plaquette) or 4 (paper layout), blocks[n-1].c_out = 4, widths that meet;
 * PD_ERR_INVALID_ARG otherwise (and for a weight count other than
 * predecoder_resnet_weight_count). */
pd_status predecoder_create_resnet(const float* weights, size_t n_weights, int32_t d, int32_t T,
                                   const pd_block* blocks, int32_t n_blocks, int32_t dtype,
                                   int32_t max_batch, const pd_options* opts, pd_predecoder** out);

/* ---- Temporal windows over a long stream (Sec. VI, parallel windows in
 * time, after the parallel-window scheme the paper cites) ----
 *
 * A stream of n_rounds rounds is cut into windows: window k commits the core
 * rounds [k core, min((k+1) core, n_rounds)) and also reads `buffer` rounds
 * before and after them (clipped to the stream).  The pre-decoder is local:
 * an output more than its receptive-field half-width h = sum over layers of
 * (k - 1) / 2 rounds from a window edge equals the output of one run over the
 * whole stream, so with buffer >= h the stitched cores are the whole-stream
 * corrections (up to the rounding-order rule of the handle's precision).  The
 * paper uses core = buffer = d (d x d x 3d blocks).  Windows are run as one
 * batch per window length (all windows of all streams at once: the paper
 * decodes the commit and cleanup blocks concurrently on several GPUs, or
 * several per GPU with a larger batch); the residual is then computed once
 * over the stitched flips of the whole stream. */
typedef struct pd_stream pd_stream; /* opaque */

/* The window plan (host only): fills starts / lengths / core_starts /
 * core_lengths (capacity entries each) and returns the number of windows,
 * ceil(n_rounds / core); with NULL arrays returns that number only.  -1 for
 * n_rounds < 1, core < 1, buffer < 0 or a capacity below the count. */
int32_t predecoder_stream_windows(int32_t n_rounds, int32_t core, int32_t buffer, int32_t* starts,
                                  int32_t* lengths, int32_t* core_starts, int32_t* core_lengths,
                                  int32_t capacity);

/* A driver for n_streams streams (independent logical qubits) of n_rounds
 * rounds at distance d: the arguments of predecoder_create_ex (weights
 * copied; the same precisions, layouts and shapes), plus the window plan.
 * opts->first_round / last_round apply to the windows at the stream's ends.
 * Creates one handle per window length; allocates device memory. */
pd_status predecoder_stream_create(const float* weights, size_t n_weights, int32_t d, int32_t n_rounds,
                                   int32_t core, int32_t buffer, const pd_layer* layers, int32_t n_layers,
                                   int32_t dtype, int32_t n_streams, const pd_options* opts, pd_stream** out);

/* det: device, [n_streams][W_det(d, n_rounds)] uint64 packed detectors;
 * flips: device, [n_streams][W_flip(d, n_rounds)], the stitched corrections;
 * residual: device, [n_streams][W_det(d, n_rounds)], the residual of the
 * whole stream from them.  Asynchronous on hip_stream. */
pd_status predecoder_stream_run(pd_stream* s, void* hip_stream, const uint64_t* det, uint64_t* flips,
                                uint64_t* residual);

/* Releases the driver (NULL is a no-op); waits for the device. */
void predecoder_stream_destroy(pd_stream* s);

/* ---- Measurement aids ----
 *
 * The ceilings the roofline fractions are quoted against, measured on the
 * device at hand (the paper times its engines on its own GPUs, Sec. VI, GPU
 * runtimes; the published MI355X peaks are the reference here).  The caller
 * times them with events on hip_stream.
 *
 * predecoder_peak_mfma: n_workgroups workgroups of four waves, each wave
 * issuing iters x 4 back-to-back matrix instructions (four independent
 * accumulators) on register operands: v_mfma_f32_32x32x16_bf16 for
 * PD_DTYPE_BF16 (32768 FLOP each), the 32x32x64 E4M3 instruction for
 * PD_DTYPE_FP8 (131072 FLOP each).  operands: device, 4096 bytes; lane l of
 * every wave takes its A operand from bytes [64 l, 64 l + 32) and its B
 * operand from [64 l + 32, 64 l + 64) (bf16: the first 16 of each); all
 * zero or random values give the two ends of the power-limited clock.  out:
 * device, n_workgroups x 256 floats (one sum per lane, so no instruction is
 * dead).  PD_ERR_INVALID_ARG for null pointers, iters or n_workgroups < 1, or
 * another dtype.  Asynchronous on hip_stream. */
pd_status predecoder_peak_mfma(void* hip_stream, int32_t dtype, const void* operands, int32_t iters,
                               int32_t n_workgroups, float* out);

/* predecoder_peak_copy: dst[0, bytes) = src[0, bytes), device buffers that
 * do not overlap, bytes a nonzero multiple of 16 (one 16-byte load and
 * store per lane): reads and writes `bytes` each.  PD_ERR_INVALID_ARG
 * otherwise.  Asynchronous on hip_stream. */
pd_status predecoder_peak_copy(void* hip_stream, const void* src, void* dst, size_t bytes);

#ifdef __cplusplus
}
#endif

#endif /* PREDECODER_H */
