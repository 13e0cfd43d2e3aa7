/*
 * hapi.h -- C ABI of the MI355X split feature-extraction library (libhapi.so).
 *
 * The library runs the storage-side half of split transfer learning: the
 * forward pass of a frozen CNN or ViT feature extractor from the input images
 * up to a chosen split layer (paper: Design and Implementation, "Request
 * flow", where the storage tier computes the frozen layers as far as the
 * requested split and returns their output; and System implementation, whose
 * models can run any contiguous range of layers), plus the per-layer output-size and forward-time profile
 * that split selection consumes (Design, "Profiling and modeling runtime" and
 * Table 1: output sizes from a batch-1 pass scale linearly with the batch;
 * the server-side forward pass is a profiled phase).
 *
 * Conventions shared by every entry point
 *  - Every data pointer is a DEVICE pointer owned by the caller (allocate with
 *    hipMalloc or as torch tensors), except the host arrays of
 *    hapi_layer_shape, hapi_profile_layers, hapi_profile_memory,
 *    hapi_stats_collect and hapi_choose_split.  The library never allocates
 *    or frees device memory; it creates hipEvents for timing and, for
 *    partitions in flight, up to 3 auxiliary streams per host thread and
 *    device.
 *  - Return value: HAPI_OK (0) or a negative hapi_status.  The message of the
 *    last failure on the calling thread is returned by hapi_last_error().
 *    Every argument is validated before anything is launched, so a call that
 *    fails validation has written nothing.
 *  - hapi_extract and hapi_pack_weights are asynchronous on desc->stream
 *    (HIP stream semantics; the caller synchronises).  hapi_profile_layers
 *    with out_us != NULL is synchronous.
 *  - Calls are reentrant given distinct streams and distinct workspaces
 *    (the paper's server runs up to 4 requests concurrently, Evaluation,
 *    Methodology).  Calls sharing a workspace must be ordered by the caller.
 *  - Results are deterministic: the same inputs give bit-identical outputs for
 *    every chunk size and across runs (frozen weights make extraction
 *    deterministic, Design, "Main insights" item 3; storage-side batch
 *    adaptation must not change results, Storage-side batch size adaptation).
 *
 * Layer numbering: layer k (1-based) is desc->layers[k-1].  A residual block or
 * transformer encoder block is one layer and ReLU / inference batch-norm belong
 * to their convolution (paper, Measurement study: a block counts as one layer
 * and only block boundaries are split points).  Split k means "the output of
 * layer k"; split 0 is the input itself (Algorithm 1 ranges the split over
 * [0, freeze index]; split 0 sends the raw input).
 */
#ifndef HAPI_H
#define HAPI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HAPI_OK = 0,
  HAPI_E_INVAL = -1,       /* bad argument: null pointer, split out of range, bad shape */
  HAPI_E_UNSUPPORTED = -2, /* a layer kind / dtype / shape combination not built */
  HAPI_E_NOMEM = -3,       /* workspace smaller than hapi_workspace_bytes() requires;
                              hapi_choose_split: even the freeze split would OOM */
  HAPI_E_DEVICE = -4       /* a HIP call or kernel launch failed */
} hapi_status;

typedef enum { HAPI_F32 = 0, HAPI_BF16 = 1 } hapi_dtype;

/* Layer kinds and the fields each one reads (others must be 0).
 *
 * HAPI_CONV        cin, cout, k, stride, pad, has_bias, has_bn, relu.
 *                  y = [ReLU]( BN( W * x + b ) ), zero padding, floor-mode size.
 * HAPI_MAXPOOL     k, stride, pad: window max, padding counts as -infinity.
 * HAPI_AVGPOOL     k == 0: global mean over H x W (output C x 1 x 1);
 *                  k > 0: k x k window mean with the given stride, no padding.
 * HAPI_BASIC_BLOCK cin, cout, stride:  ReLU(bn2(conv2(ReLU(bn1(conv1(x))))) + sc(x)),
 *                  conv1 3x3/stride, conv2 3x3/1, sc = bn(conv1x1/stride) when
 *                  stride != 1 or cin != cout, else identity.
 * HAPI_BOTTLENECK  cin, width, stride:  ReLU(c3(c2(c1(x))) + sc(x)) with
 *                  c1 1x1 cin->width, c2 3x3/stride width->width, c3 1x1
 *                  width->4*width, each with BN (ReLU after c1, c2); sc as above.
 * HAPI_PATCH_EMBED cin, cout (= model width D), k (= patch size, also the stride):
 *                  non-overlapping patch projection with bias, no activation.
 * HAPI_TOKENS      cout (= D): [N, D, h, w] -> [N, 1 + h*w, D]; patch t = row*w + col
 *                  becomes token 1 + t, a class token is token 0, and the
 *                  position embedding is added to every token.
 * HAPI_VIT_BLOCK   cout (= D), heads, mlp_dim: pre-norm encoder block
 *                  x += out_proj(MHA(LN1(x))); x += fc2(GELU(fc1(LN2(x)))),
 *                  layernorm eps 1e-6, exact-erf GELU, softmax(QK^T/sqrt(D/heads))V.
 * HAPI_LAYERNORM   cout (= D): per-token layernorm with affine, eps 1e-6.
 * HAPI_DENSE_BLOCK cin, cout (= cin + n * growth), width (= growth), mlp_dim
 *                  (= bottleneck channels): DenseNet dense block of n layers;
 *                  layer l maps the c = cin + l * growth channels so far to
 *                  conv3x3(ReLU(BN2(conv1x1(ReLU(BN1(x)))))) (growth channels,
 *                  pad 1) and concatenates them after the existing channels.
 * HAPI_PREACT_CONV cin, cout, k, stride, pad: pre-activation convolution
 *                  y = W * ReLU(BN(x)), no bias (DenseNet transition; the
 *                  batch-norm acts on the input, so it cannot fold into W).
 * HAPI_BATCHNORM   cout (= channels), relu: y = [ReLU](BN(x)) per channel.
 *
 * Batch-norm is inference-mode with eps 1e-5. */
typedef enum {
  HAPI_CONV = 0,
  HAPI_MAXPOOL = 1,
  HAPI_AVGPOOL = 2,
  HAPI_BASIC_BLOCK = 3,
  HAPI_BOTTLENECK = 4,
  HAPI_PATCH_EMBED = 5,
  HAPI_TOKENS = 6,
  HAPI_VIT_BLOCK = 7,
  HAPI_LAYERNORM = 8,
  HAPI_DENSE_BLOCK = 9,
  HAPI_PREACT_CONV = 10,
  HAPI_BATCHNORM = 11
} hapi_kind;

typedef struct {
  int32_t kind;                       /* hapi_kind */
  int32_t cin, cout, width;           /* channels (width: bottleneck inner width) */
  int32_t k, stride, pad;             /* window / kernel geometry */
  int32_t relu, has_bias, has_bn;     /* HAPI_CONV options (0/1) */
  int32_t heads, mlp_dim;             /* HAPI_VIT_BLOCK */
  int32_t reserved[4];                /* must be 0 */
} hapi_layer;

typedef struct {
  int32_t n_layers;                   /* >= 1 */
  const hapi_layer *layers;           /* host array of n_layers entries */
  int32_t dtype;                      /* hapi_dtype of images, activations and outputs */
  int32_t in_c, in_h, in_w;           /* per-image input shape (NCHW) */
  void *stream;                       /* hipStream_t; NULL = the null stream */
  void *workspace;                    /* device scratch owned by the caller */
  size_t workspace_bytes;
  int32_t chunk;                      /* storage-side (COS) batch: images per partition;
                                         0 = the library chooses */
  int32_t inflight;                   /* partitions in flight at once, 0..4; 0 = the
                                         library chooses: 2 when chunk == 0 and the
                                         batch has >= 128 images, else 1 (sequential) */
  int32_t direct;                     /* 0: repeated identical extractions replay a
                                         captured HIP graph (see hapi_extract);
                                         1: every call launches its kernels one by one */
} hapi_model_desc;

/* Raw (unpacked) weights: ONE flat float32 device buffer holding, layer by
 * layer in order, the PyTorch-layout tensors below (nothing for pools):
 *   CONV         weight [cout, cin, k, k]; bias [cout] if has_bias;
 *                gamma, beta, running_mean, running_var [cout] each if has_bn
 *   BASIC_BLOCK  conv1 weight, bn1 (4 x [cout]); conv2 weight, bn2;
 *                shortcut weight [cout, cin, 1, 1], shortcut bn (only if present)
 *   BOTTLENECK   conv1 weight [width, cin, 1, 1], bn1; conv2 weight
 *                [width, width, 3, 3], bn2; conv3 weight [4w, width, 1, 1], bn3;
 *                shortcut weight + bn (only if present)
 *   PATCH_EMBED  weight [D, cin, k, k], bias [D]
 *   TOKENS       class token [D], position embedding [T, D] (T = 1 + h*w)
 *   VIT_BLOCK    ln1 gamma, beta [D]; in-proj weight [3D, D] (rows: query, key,
 *                value), bias [3D]; out-proj weight [D, D], bias [D]; ln2 gamma,
 *                beta [D]; fc1 weight [mlp, D], bias [mlp]; fc2 weight [D, mlp], bias [D]
 *   LAYERNORM    gamma, beta [D]
 *   DENSE_BLOCK  per dense layer l (c = cin + l * growth): bn1 gamma, beta, mean,
 *                var [c]; conv1 weight [bottleneck, c, 1, 1]; bn2 gamma, beta,
 *                mean, var [bottleneck]; conv2 weight [growth, bottleneck, 3, 3]
 *   PREACT_CONV  bn gamma, beta, mean, var [cin]; weight [cout, cin, k, k]
 *   BATCHNORM    gamma, beta, mean, var [cout]
 * Returns the number of float32 values, or a negative hapi_status. */
int64_t hapi_raw_weight_count(const hapi_model_desc *desc);

/* Bytes of the packed-weight buffer hapi_pack_weights writes, or < 0 on error. */
int64_t hapi_packed_weight_bytes(const hapi_model_desc *desc);

/* Model load (the "read model to GPU" phase of Table 1): folds inference
 * batch-norm into the preceding convolution in float32 (W' = W g/sqrt(v+eps),
 * b' = beta + (b - mean) g/sqrt(v+eps)), reorders convolution weights for the
 * kernels and casts them to desc->dtype.  raw_weights: device float32 buffer of
 * hapi_raw_weight_count() values (layout above); packed: device buffer of
 * hapi_packed_weight_bytes() bytes, 256-byte aligned.  Packed weights are
 * reused by any number of hapi_extract calls (model reuse, Design, "Request
 * flow").  Asynchronous on desc->stream; needs no workspace. */
int hapi_pack_weights(const hapi_model_desc *desc, const void *raw_weights, void *packed);

/* Per-image output shape of layer `layer` (0 = input) in the caller layout:
 * NCHW {C, H, W} for convolutional layers (ndim 3), {T, D} for token layers
 * (ndim 2).  dims must hold 3 values.  Host only. */
int hapi_layer_shape(const hapi_model_desc *desc, int32_t layer, int64_t *dims, int32_t *ndim);

/* Workspace bytes hapi_extract(batch, split_layer) needs with desc->chunk
 * (profile != 0: what hapi_profile_layers(batch, out_us != NULL) needs, which
 * also holds synthetic weights and inputs).  At least the paper's memory
 * estimate -- the largest input + output of any layer at the chunk batch
 * (Design, "Memory usage estimation"; over-estimating is the safe side) --
 * plus block-internal temporaries.  Returns bytes or a negative hapi_status. */
int64_t hapi_workspace_bytes(const hapi_model_desc *desc, int32_t batch, int32_t split_layer,
                             int32_t profile);

/* Guard gaps of the workspace hapi_extract uses for (batch, split_layer)
 * with desc->chunk and desc->inflight: each of the library's workspace
 * regions (three activation slots and a partial-sum region per partition in
 * flight) is followed by HAPI_GUARD_BYTES that no kernel writes.  Writes the
 * byte offsets of the gaps, relative to desc->workspace, into
 * offsets[0 .. min(count, max_entries)) and returns their count (0 for split
 * 0), or a negative hapi_status.  For checking kernels' bounds: fill the gaps
 * with a pattern before a call, compare them after it.  Host only. */
#define HAPI_GUARD_BYTES 4096
int32_t hapi_workspace_guards(const hapi_model_desc *desc, int32_t batch, int32_t split_layer,
                              int64_t *offsets, int32_t max_entries);

/* Number of partitions (storage-side batches) hapi_extract uses for `batch`
 * images with desc->chunk (Storage-side batch size adaptation: a request is
 * processed as partitions of the storage-side batch; the last partition may
 * be short).  Host only; < 0 on error. */
int32_t hapi_chunk_count(const hapi_model_desc *desc, int32_t batch);

/* Partitions in flight.  With k = min(inflight, partitions) > 1, partition p
 * runs on lane p % k: lane 0 is desc->stream, lanes 1..k-1 are auxiliary
 * streams (default priority) that the library creates once per host thread
 * and device, forks from desc->stream at the start of the call and joins back
 * into it at the end, so the call stays asynchronous and ordered on
 * desc->stream.  Each lane has its own workspace slots (the workspace grows
 * with k).  The paper's server runs up to 4 requests at once (Evaluation,
 * Methodology); on this GPU partitions in flight overlap each other's layer
 * ramps and tails.  Results do not depend on chunk or inflight. */

/* The storage-side forward pass.
 *   weights      packed weights from hapi_pack_weights (same desc)
 *   images       [batch, in_c, in_h, in_w] NCHW in desc->dtype
 *   batch        >= 1 images
 *   split_layer  0..n_layers: layers 1..split_layer run; 0 copies the input
 *   out          [batch, <hapi_layer_shape(split_layer)>] in desc->dtype,
 *                NCHW for convolutional layers, [batch, T, D] for token
 *                layers; row i always belongs to image i
 * The batch runs as hapi_chunk_count() sequential partitions through the
 * workspace.  Errors: HAPI_E_INVAL (null pointer, batch < 1, split out of
 * range), HAPI_E_NOMEM (workspace too small), HAPI_E_UNSUPPORTED,
 * HAPI_E_DEVICE (a launch failed).  Asynchronous on desc->stream.
 *
 * Plan replay (desc->direct == 0).  A call identical to the previous
 * extraction on the same host thread (same layers, dtype, input shape, chunk,
 * inflight, device, pointers, batch and layer range) is captured once as a
 * HIP graph -- every kernel launch of the call with its fork and join of the
 * auxiliary streams -- and the graph is launched on desc->stream; later
 * identical calls launch that graph again (the library keeps the 8 most
 * recent graphs per host thread until the process ends).  The graph runs the
 * same kernels with the same arguments, so results are bit-identical to
 * direct launches; it only removes the per-kernel launch cost (which bounds
 * small batches; Storage-side batch size adaptation asks throughput to hold
 * at every batch).  A graph reads the pointers it was captured with: contents
 * may change between calls, buffers must not be freed while a call that
 * uses them is pending (as with direct launches).  Calls made while kernel
 * statistics are enabled always launch directly.  The graph has no memset
 * nodes. */
int hapi_extract(const hapi_model_desc *desc, const void *weights, const void *images,
                 int32_t batch, int32_t split_layer, void *out);

/* hapi_extract for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same arguments and results as hapi_extract (bit-identical outputs), but
 * desc->workspace and desc->workspace_bytes are ignored and the library's own
 * device scratch is used instead -- a static array of
 * HAPI_NOALLOC_SCRATCH_BYTES per GPU, part of the library's code object,
 * held by each GPU the library runs on until the process ends.  The call
 * allocates nothing (no hipMalloc/hipFree, no stream, event or graph
 * creation): its partitions run one after another on desc->stream, with
 * direct kernel launches.  The first call on a device, with that device
 * current, looks up the scratch's address on it.
 *   Errors: as hapi_extract; HAPI_E_NOMEM when the extraction needs more
 *   than HAPI_NOALLOC_SCRATCH_BYTES of workspace (hapi_workspace_bytes with
 *   desc->inflight = 1 tells how much; lower the batch or desc->chunk);
 *   HAPI_E_INVAL when desc->stream is not on the current device.
 *   Every call on one GPU shares that GPU's scratch: calls that overlap on a
 *   GPU (different streams or host threads) race and give wrong results;
 *   order them.  Nothing in the scratch needs to start at zero (every region
 *   is written before it is read), so the contents a previous call left do
 *   not matter. */
#define HAPI_NOALLOC_SCRATCH_BYTES ((int64_t)256 << 20)
int hapi_extract_noalloc(const hapi_model_desc *desc, const void *weights, const void *images,
                         int32_t batch, int32_t split_layer, void *out);

/* Resume from a split (the compute-tier half: System implementation, models
 * that run the forward pass between arbitrary layers; Design, "Request flow",
 * the client continues from the split layer's output).  Runs layers
 * start_layer+1 .. end_layer on
 *   input   [batch, <hapi_layer_shape(start_layer)>] in desc->dtype, the
 *           caller layout hapi_extract writes (NCHW or [batch, T, D])
 * and writes out as hapi_extract(end_layer) does.  0 <= start_layer <=
 * end_layer <= n_layers; start_layer = 0 is hapi_extract, start_layer =
 * end_layer copies the input.  The same kernels and rounding points run as in
 * a single pass, so hapi_extract(s) followed by hapi_extract_range(s, e) gives
 * hapi_extract(e) bit for bit.  Workspace: hapi_workspace_bytes(desc, batch,
 * end_layer, 0).  Errors and stream semantics as hapi_extract. */
int hapi_extract_range(const hapi_model_desc *desc, const void *weights, const void *input,
                       int32_t batch, int32_t start_layer, int32_t end_layer, void *out);

/* Per-layer profile for split selection (Table 1; Measurement study, Fig. 2a/2b).
 *   out_bytes[k], k = 0..n_layers: bytes of the layer-k output at `batch`
 *                 (k = 0: the input), closed form, no device access.
 *   out_us[k]:    device time in microseconds of layer k at `batch` with
 *                 desc->chunk, median of 20 timed passes after 5 warm-ups, on
 *                 synthetic weights and inputs written into the workspace
 *                 (out_us[0] = 0).  NULL skips timing; then the call touches
 *                 no device and works without a GPU.
 * The partitions hapi_extract would use run one after another on
 * desc->stream, each layer bracketed by events, with the tile choice
 * hapi_extract makes for the same batch (which depends on the partitions it
 * keeps in flight), so the kernels timed are the ones an extraction runs; the
 * ResNet stem and its max pooling, fused in an extraction, are timed as the
 * two layers they are.  With one partition in flight the sum over layers
 * approximates an extraction's time; with several, it exceeds it by the
 * overlap of the partitions.
 * Synchronous.  With out_us the workspace must hold
 * hapi_workspace_bytes(desc, batch, n_layers, 1) bytes. */
int hapi_profile_layers(const hapi_model_desc *desc, int32_t batch, int64_t *out_bytes,
                        float *out_us);

/* Per-split device memory (Measurement study, Fig. 2c: per-layer peak GPU
 * memory).  bytes[k], k = 0..n_layers: every device byte a hapi_extract of
 * `batch` images to split k uses with desc->chunk -- the packed weights of
 * layers 1..k (a packed buffer for the first k layers is exactly that
 * prefix), the images, the output and the workspace; the library allocates
 * nothing else.  Host only, closed form, works without a GPU. */
int hapi_profile_memory(const hapi_model_desc *desc, int32_t batch, int64_t *bytes);

/* Per-kernel timing of later hapi_extract calls (for roofline reporting).
 * hapi_stats_enable(1) clears the counters and brackets every kernel launch of
 * hapi_extract with HIP events on desc->stream; hapi_stats_enable(0) stops.
 * hapi_stats_collect synchronises the recorded events and fills up to
 * `max_entries` rows, one per kernel family, returning the number of families
 * (or < 0).  flops / bytes are the algorithmic counts of the recorded launches. */
typedef struct {
  char name[32];
  int64_t launches;
  double total_ms;    /* sum of the launches' durations */
  double flops;
  double bytes;
  double busy_ms;     /* time at least one launch of the family was running (differs
                         from total_ms when partitions in flight overlap) */
} hapi_kernel_stat;

int hapi_stats_enable(int32_t enable);
int hapi_stats_collect(hapi_kernel_stat *out, int32_t max_entries);

/* ---------------------------------------------------------------------------
 * Split-index choice (Algorithm 1 and its competitors, Evaluation,
 * Methodology).  Pure host arithmetic over the profile above plus the
 * caller's client-side and environment measurements; no device access, works
 * without a GPU.  Times in seconds, sizes in bytes.
 *
 * Per-iteration estimates for a split s (phases of Table 1; "Profiling and
 * modeling runtime"):
 *   requests  R = train_batch / request_images, waves V = ceil(R / server_slots)
 *   RT_SRV(s) = V * [read_data + read_model + to_gpu
 *                    + request_images * image_bytes[s] * (from_gpu + pickle)]
 *               + R * sum_{k=1..s} srv_layer_s[k]
 *     (the forward passes of concurrent requests serialise on the GPU, every
 *     other phase runs in parallel, and a request waits for the wave of
 *     requests in front of it).  At s = 0 the server runs no layer: only
 *     read_data and pickle remain.
 *   RT_NW(s)  = train_batch * image_bytes[s] / net_bytes_per_s
 *   RT_CLI(s) = train_batch * image_bytes[s] * (unpickle + loader + cli_to_gpu)
 *               + sum_{k=s+1..n_layers} cli_layer_s[k] + cli_rest_s
 *   memory(s) = cli_fixed_mem_bytes + train_batch * max(image_bytes[s],
 *               max_{k=s+1..n_layers} (image_bytes[k-1] + image_bytes[k]))
 *     (Design, "Memory usage estimation": the peak of the forward pass is the
 *     layer with the largest input + output); s is predicted to OOM when
 *     cli_mem_bytes > 0 and memory(s) > cli_mem_bytes.
 *   epoch(s)  = RT_SRV + max(RT_SRV + RT_NW, RT_CLI) * (iterations - 1) + RT_CLI
 *     (Algorithm 1: the client's work overlaps the server's work and the
 *     transfer of the next iteration).  When nosplit_iter_s > 0, split 0 uses
 *     iterations * nosplit_iter_s instead: its per-iteration time was measured
 *     while profiling the earliest split (Design, notes after Algorithm 1).
 * Sums over layers run in ascending k; argmins take the earliest index on ties.
 */
typedef struct {
  int32_t n_layers;           /* layers of the profiled model, >= 1 */
  int32_t freeze_idx;         /* user's freeze index, 0..n_layers */
  int32_t train_batch;        /* training batch size (images per iteration), >= 1 */
  int32_t request_images;     /* images per POST request (paper: 128); divides train_batch */
  int32_t server_slots;       /* requests the server runs at once (paper: 4), >= 1 */
  int32_t reserved0;          /* must be 0 */
  int64_t iterations;         /* NR_IT: iterations per epoch, >= 1 */
  const int64_t *image_bytes; /* [n_layers+1] host: layer-k output bytes of ONE image
                                 (hapi_profile_layers at batch 1), each >= 1 */
  const double *srv_layer_s;  /* [n_layers+1] host: server forward time of layer k for one
                                 request (hapi_profile_layers out_us at batch
                                 request_images, in seconds); [0] is ignored */
  const double *cli_layer_s;  /* [n_layers+1] host: client forward time of layer k at the
                                 training batch; [0] is ignored */
  double srv_read_data_s;     /* per request: read its objects from storage */
  double srv_read_model_s;    /* per request: load the model to the GPU (0 with reuse) */
  double srv_to_gpu_s;        /* per request: move its input to the GPU */
  double cli_rest_s;          /* per iteration: split-independent client work (layers after
                                 the profiled ones, backward pass, optimiser step) */
  double srv_from_gpu_s_per_byte; /* linear phases, seconds per byte of split output */
  double srv_pickle_s_per_byte;
  double cli_unpickle_s_per_byte;
  double cli_loader_s_per_byte;
  double cli_to_gpu_s_per_byte;
  double net_bytes_per_s;     /* network bandwidth, > 0 */
  int64_t cli_mem_bytes;      /* client GPU memory; 0 = never predict an OOM */
  int64_t cli_fixed_mem_bytes;/* split-independent client memory (weights, optimiser,
                                 training activations) */
  double nosplit_iter_s;      /* measured per-iteration time at split 0, or <= 0 */
} hapi_split_job;

typedef struct {
  double rt_srv, rt_nw, rt_cli; /* per-iteration estimates */
  double epoch_s;               /* Algorithm 1's epoch runtime estimate */
  double sum_s;                 /* RT_SRV + RT_NW + RT_CLI (NSG's objective) */
  int64_t cli_mem_bytes;        /* client memory estimate */
  int32_t oom;                  /* 1 = predicted to run out of client memory */
  int32_t reserved;
} hapi_split_estimate;

typedef struct {
  int32_t hapi;       /* Algorithm 1: argmin epoch_s over non-OOM splits in [0, freeze_idx] */
  int32_t earliest;   /* earliest non-OOM split (profiled in the second half of epoch 0) */
  int32_t freeze;     /* @Freeze: freeze_idx */
  int32_t min_output; /* @Min: smallest image_bytes[k] over k = 1..freeze_idx, earliest
                         on ties (0 when freeze_idx = 0); may be predicted to OOM */
  int32_t nosplit;    /* NoSplit: 0; may be predicted to OOM */
  int32_t nsg;        /* NSG: argmin sum_s over non-OOM splits in [0, freeze_idx] */
} hapi_split_choice;

/* Fills `choice` and, if `est` is not NULL, est[s] for s = 0..freeze_idx (host
 * arrays owned by the caller).  Errors: HAPI_E_INVAL (NULL pointer, a count or
 * index out of range, a negative or non-finite time or rate, train_batch not
 * a multiple of request_images, a byte count that overflows), HAPI_E_NOMEM
 * (the freeze split itself is predicted to OOM: so is every other split,
 * Algorithm 1's first step).  On error nothing is written. */
int hapi_choose_split(const hapi_split_job *job, hapi_split_estimate *est,
                      hapi_split_choice *choice);

/* Message of the last failed call on this thread ("" if none). */
const char *hapi_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* HAPI_H */
