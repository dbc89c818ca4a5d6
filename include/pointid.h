/*
 * pointid.h — C ABI of libpointid: per-hit track / shower / Michel
 * classification on one AMD Instinct MI355X (gfx950).
 *
 * The operation (paper §2.1 and §2.3): for every reconstructed wire hit, given
 * by its wire number and peak time, a 48x48 patch is cut from the plane's
 * deconvolved charge image, rows indexing the wire and columns the time, and
 * classified by the CNN of paper §2.2 — 48 filters of 5x5 at stride 1 (48 maps
 * of 44x44) with ReLU, a 128-neuron and a 32-neuron fully connected layer with
 * ReLU, then a 3-output softmax branch and a 1-output sigmoid (Michel) branch.
 *
 * Readings of the paper fixed by this ABI:
 *   - patch pixel (r, c) of hit (w, t) is image[w - 24 + r][t - 24 + c]; any
 *     pixel outside the plane reads 0 (so the hit sits at pixel (24, 24));
 *   - one image column is one time tick; the image is not rescaled;
 *   - the filter is a cross-correlation (no flip); the maps are flattened
 *     channels-last, FC1 input index (y*44 + x)*48 + k;
 *   - dropout is the identity at inference.
 *
 * Conventions for every entry point:
 *   - All pointers named image/hits/patches/scores are DEVICE pointers on the
 *     handle's device, owned by the caller, who keeps them alive until the
 *     stream has passed the call.  Weight pointers are HOST pointers.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Calls
 *     only enqueue work on it; none synchronises the host.  Temporary device
 *     memory comes from scratch buffers the handle caches until
 *     pointid_destroy: a call takes a free buffer that its stream last used or
 *     whose last use has finished (else it makes `stream` wait for that use),
 *     so calls after the first few allocate nothing; a call allocates
 *     (hipMalloc) only when no cached buffer is free and big enough.
 *   - A handle is immutable after pointid_create: any number of host threads
 *     and streams may use one handle at once.
 *   - Results are deterministic: identical inputs give identical bits, and
 *     permuting the hits permutes the scores bit for bit (no atomics, fixed
 *     reduction order).
 *   - Status codes are returned; arguments are validated on the host before any
 *     launch; no C++ exception crosses the ABI.  On a non-OK status,
 *     pointid_last_error() returns a description for the calling thread.
 *   - n == 0 is a successful no-op (no launch, pointers may be NULL).
 *   - Hit coordinates are never errors: pixels outside their plane read 0,
 *     whole patches included; a plane index out of range gives an all-zero
 *     patch.  Inputs must be finite (not checked).
 */
#ifndef POINTID_H
#define POINTID_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
enum {
    POINTID_OK = 0,
    POINTID_EINVAL = -1,        /* bad argument (NULL pointer, negative size, ...) */
    POINTID_ENOMEM = -2,        /* device allocation failed */
    POINTID_EHIP = -3,          /* a HIP runtime call or kernel launch failed */
    POINTID_ENODEV = -4,        /* no usable gfx950 device */
    POINTID_EUNSUPPORTED = -5,  /* precision or dtype not supported */
    POINTID_EIO = -6            /* socket I/O failed or the peer closed (server / client) */
};

/* arithmetic of a handle (pointid_create) or element type of a patch buffer */
enum {
    POINTID_FP32 = 0,           /* fp32 inputs, weights, accumulation */
    POINTID_BF16 = 1,           /* bf16 patch, conv filter, conv output and FC1
                                   filter (round to nearest even); fp32
                                   accumulation, biases, FC2 and heads */
    POINTID_FP16 = 2,           /* as POINTID_BF16 with IEEE fp16 operands:
                                   same MFMA rate, 3 more mantissa bits; a conv
                                   output above 65504 in magnitude overflows */
    POINTID_FP8 = 3             /* handles only (paper §4: 8-bit operation):
                                   the conv as POINTID_FP16; its ReLU output
                                   (clamped to 448) and the FC1 filter rounded
                                   to OCP e4m3, FC1 column n first multiplied
                                   by 2^k_n, the largest power of two keeping
                                   the column within 448, and its sums by
                                   2^-k_n; fp32 accumulation, biases, FC2 and
                                   heads.  Patches are made in fp16. */
};

/* Patch and network shape, paper §2.1-§2.2. */
#define POINTID_PATCH 48
#define POINTID_KSIZE 5
#define POINTID_NCH 48
#define POINTID_FMAP 44
#define POINTID_FC1_IN 92928     /* 44 * 44 * 48 */
#define POINTID_FC1_OUT 128
#define POINTID_FC2_OUT 32
#define POINTID_NCLS 3
#define POINTID_NSCORES 4        /* (p_track, p_em, p_none, p_michel) */
#define POINTID_MAX_PLANES 64

typedef struct pointid_s *pointid_handle;

/*
 * Host fp32 weights of the network of paper §2.2 (11,900,420 values), all
 * C-contiguous, owned by the caller and only read during pointid_create.
 */
typedef struct {
    const float *conv_w;   /* [48][5][5]: filter k, u = wire offset, v = tick offset */
    const float *conv_b;   /* [48] */
    const float *fc1_w;    /* [92928][128]: row (y*44 + x)*48 + k */
    const float *fc1_b;    /* [128] */
    const float *fc2_w;    /* [128][32] */
    const float *fc2_b;    /* [32] */
    const float *cls_w;    /* [32][3]  softmax branch */
    const float *cls_b;    /* [3] */
    const float *mic_w;    /* [32]     sigmoid (Michel) branch */
    const float *mic_b;    /* [1] */
} pointid_weights;

/* One plane of a multi-plane call: device fp32 image [n_wires][n_ticks],
 * tick fastest (row pitch n_ticks floats). */
typedef struct {
    const float *image;
    int32_t n_wires;
    int32_t n_ticks;
} pointid_plane;

/*
 * Create a classifier on `device` (HIP ordinal) computing in `precision`
 * (POINTID_FP32, POINTID_BF16, POINTID_FP16 or POINTID_FP8).  The weights are
 * converted and repacked into device memory owned by the handle (POINTID_FP8:
 * the per-column exponents k_n are taken from the fp32 FC1 weights on the
 * host; the factor 2^-k_n is an fp32 value, subnormal for a column whose
 * largest magnitude is below 2^-118 and zero below 2^-141); the call is
 * synchronous, so the host weights may be freed when it returns.
 * Errors: EINVAL (NULL w, NULL member, NULL out), EUNSUPPORTED (precision),
 * ENODEV (no such device, or not gfx950), ENOMEM, EHIP.  *out is set to NULL
 * on failure.
 */
int pointid_create(const pointid_weights *w, int precision, int device,
                   pointid_handle *out);

/* Free a handle (synchronises its device first).  NULL is a no-op. */
int pointid_destroy(pointid_handle h);

/*
 * Free cached scratch buffers (see "Temporary device memory" above) until the
 * handle caches at most `keep_bytes`, largest buffers first.  Only idle
 * buffers are freed: none that a call on another thread is taking, and none
 * whose last user's work is still running (those stay cached; call again
 * later).  keep_bytes = 0 frees every idle buffer.  The next call that needs
 * scratch allocates again.  hipFree may wait for the device.  The cache holds
 * at most 512 buffers in any case; when they are all taken, a call reuses the
 * smallest one big enough and waits on its stream for that buffer's last use.
 *   cached_bytes  (optional, may be NULL) receives the bytes still cached
 * Errors: EINVAL (NULL handle), EHIP (hipFree failed; the buffers freed before
 * the failure stay freed).
 */
int pointid_trim(pointid_handle h, uint64_t keep_bytes, uint64_t *cached_bytes);

/* Precision the handle was created with, or EINVAL for NULL. */
int pointid_precision(pointid_handle h);

/*
 * Classify hits of one plane (paper §2.3: the module passes each hit's wire
 * number and peak time; the patch is built and classified).
 *   image  device fp32 [n_wires][n_ticks]
 *   hits   device int32 [n_hits][2] = (wire, tick)
 *   scores device fp32 [n_hits][4] = (p_track, p_em, p_none, p_michel), written
 *          in hit order; the first three sum to 1 (softmax), the last is the
 *          sigmoid output.  16-byte aligned.
 * Errors: EINVAL (NULL handle; n_hits < 0; n_wires or n_ticks <= 0; NULL
 * pointer with n_hits > 0; misaligned scores), ENOMEM (workspace), EHIP
 * (launch).
 */
int pointid_classify(pointid_handle h, const float *image, int32_t n_wires,
                     int32_t n_ticks, const int32_t *hits, int64_t n_hits,
                     float *scores, void *stream);

/*
 * Classify hits spread over several planes in one call (an event, paper §2.1:
 * data are processed per wire plane).
 *   planes  HOST array of n_planes descriptors (1 <= n_planes <= 64), read
 *           during the call only
 *   hits    device int32 [n_hits][3] = (plane, wire, tick)
 *   scores  device fp32 [n_hits][4], in hit order
 * Errors as pointid_classify, plus EINVAL for n_planes out of range or a plane
 * with a NULL image or non-positive size.
 */
int pointid_classify_planes(pointid_handle h, const pointid_plane *planes,
                            int32_t n_planes, const int32_t *hits,
                            int64_t n_hits, float *scores, void *stream);

/*
 * pointid_classify_planes without any device allocation, for callers that
 * cannot allocate (code under HIP graph capture, tight serving loops, hosts
 * that forbid hipMalloc): the same arguments, kernels and bits, with the
 * call's scratch (patches and split-K partials) in a fixed device array of
 * the library (104 MiB per GPU, held from the first call on a GPU until the
 * process ends) instead of the handle's cache.  n_hits is at most 8192.
 * Every call on one GPU shares that array: calls that overlap on one GPU
 * (other streams or threads) race and must be ordered by the caller.  No
 * part of the array needs clearing between calls.
 * Errors as pointid_classify_planes, plus EINVAL for n_hits > 8192.
 */
int pointid_classify_planes_noalloc(pointid_handle h, const pointid_plane *planes,
                                    int32_t n_planes, const int32_t *hits,
                                    int64_t n_hits, float *scores, void *stream);

/*
 * Classify hits with patches whose columns span D = ticks_per_column ticks
 * each (paper §2.1: a pixel holds the charge its wire collects in the time
 * interval of its column).  Each plane is binned once into columns of D ticks
 * aligned to tick 0 -- column j holds the charge of ticks jD .. jD + D - 1,
 * their sum (ticks past the end of the plane count as 0), accumulated in fp64
 * and rounded to fp32 once -- and the patch of hit
 * (plane, wire, tick) is cut from the binned plane around column
 * floor(tick / D), exactly as pointid_classify_planes cuts it around a tick.
 * D = 1 gives pointid_classify_planes' bits.
 *   planes  HOST array of the unbinned planes, as in pointid_classify_planes
 *   hits    device int32 [n_hits][3] = (plane, wire, tick), ticks unbinned
 *   scores  device fp32 [n_hits][4], in hit order, 16-byte aligned
 * The binned planes (image bytes / D) live in the handle's scratch cache.
 * Errors as pointid_classify_planes, plus EINVAL for ticks_per_column < 1.
 */
int pointid_classify_planes_ds(pointid_handle h, const pointid_plane *planes,
                               int32_t n_planes, int32_t ticks_per_column,
                               const int32_t *hits, int64_t n_hits,
                               float *scores, void *stream);

/* One request of a batched call. */
typedef struct {
    const int32_t *hits;   /* device int32: [n_hits][2] = (wire, tick) on plane
                              `plane`, or [n_hits][3] = (plane, wire, tick)
                              when plane < 0 */
    int64_t n_hits;        /* >= 0; a request with no hits is skipped */
    int32_t plane;         /* index into the call's planes, or -1 */
    float *scores;         /* device fp32 [n_hits][4], 16-byte aligned */
} pointid_request;

/*
 * Classify several independent requests in one launch sequence (paper §2.3:
 * the server combines requests from many clients into larger batches, which
 * §3.2 measures with dynamic batching).  The requests' hits are classified as
 * one batch over the shared `planes`; each request's scores land in its own
 * output, with exactly the bits pointid_classify (plane >= 0) or
 * pointid_classify_planes (plane < 0) gives that request alone.  More than 64
 * non-empty requests run as consecutive batches of 64.
 *   planes    HOST array, 1 <= n_planes <= 64, read during the call only
 *   requests  HOST array of n_requests, read during the call only
 * Errors: EINVAL (NULL handle, planes or requests; n_requests < 0; a request
 * with n_hits < 0, plane >= n_planes, or a NULL or misaligned pointer with
 * n_hits > 0; a plane as in pointid_classify_planes), ENOMEM, EHIP.  Every
 * request is checked before any is classified.
 */
int pointid_classify_requests(pointid_handle h, const pointid_plane *planes,
                              int32_t n_planes, const pointid_request *requests,
                              int32_t n_requests, void *stream);

/*
 * Dynamic batching (paper §2.3; measured in §3.2): requests submitted from
 * any host threads are merged, in arrival order, into pointid_classify_requests
 * calls of at most `max_requests` (1..4096) requests over the resident
 * `planes`, issued on the batcher's own stream as soon as `max_requests` are
 * pending or the oldest has waited `max_delay_us` microseconds.  Up to 4
 * batches run at once.  A request's scores are those it gets alone, bit for
 * bit.  The handle and the plane images must outlive the batcher; a request's
 * hits and scores buffers must stay valid until its wait returns.
 * create errors: EINVAL (NULL out, handle or planes; a bad plane; n_planes,
 * max_requests or max_delay_us out of range), EHIP.
 */
typedef struct pointid_batcher_s *pointid_batcher;
int pointid_batcher_create(pointid_handle h, const pointid_plane *planes,
                           int32_t n_planes, int32_t max_requests,
                           int32_t max_delay_us, pointid_batcher *out);
/* Classify every pending request, wait for all, then free.  NULL is a no-op. */
int pointid_batcher_destroy(pointid_batcher b);
/* Queue one request (copied; its buffers are not).  *ticket identifies it.
 * `stream` (a hipStream_t on the handle's device, or NULL for the null
 * stream) orders the request after the work already enqueued there: submit
 * records an event on it, and the batch that classifies the request waits for
 * that event before reading the hits or writing the scores.  So the hits may
 * still be in production on `stream` (pointid_find_hits, a copy), and the
 * scores buffer may come from an allocator that orders reuse by `stream`.
 * Errors: EINVAL (NULL argument, bad request as in pointid_classify_requests,
 * batcher being destroyed), EHIP (the event could not be recorded on
 * `stream`). */
int pointid_batcher_submit(pointid_batcher b, const pointid_request *req,
                           void *stream, uint64_t *ticket);
/* Block until the request `ticket` is classified: its scores are then in
 * device memory, visible to the host and to every stream.  Returns the status
 * of its batch (EHIP or ENOMEM if that batch failed), or EINVAL for a ticket
 * this batcher did not issue. */
int pointid_batcher_wait(pointid_batcher b, uint64_t ticket);

/*
 * Classify pre-cut patches (the model interface of paper §2.3, which receives
 * batches of ready patches).
 *   patches device fp32 [n][48][48] (row = wire, column = tick), 16-byte aligned
 *   scores  device fp32 [n][4], 16-byte aligned
 * 16-bit and 8-bit handles round the patches to their 16-bit type first
 * (8-bit handles: fp16), inside the fused kernel for up to 4,096 patches on
 * 16-bit handles, else in a separate pass.
 * Errors: EINVAL (NULL handle, n < 0, NULL or misaligned pointer with n > 0),
 * ENOMEM, EHIP.
 */
int pointid_classify_patches(pointid_handle h, const float *patches, int64_t n,
                             float *scores, void *stream);

/*
 * Patch construction alone (paper §2.1), for checking and preprocessing; needs
 * no handle and runs on the current HIP device.
 *   patches_out device [n_hits][48][48] of fp32 (out_dtype POINTID_FP32) or
 *               bf16 / fp16 bit patterns (POINTID_BF16 / POINTID_FP16, round to
 *               nearest even),
 *               16-byte aligned; the image may have any alignment
 * Bit-exact: fp32 values are copied, never computed.
 * Errors: EINVAL, EUNSUPPORTED (out_dtype), EHIP.
 */
int pointid_gather(const float *image, int32_t n_wires, int32_t n_ticks,
                   const int32_t *hits, int64_t n_hits, void *patches_out,
                   int out_dtype, void *stream);

/* Multi-plane patch construction; hits are (plane, wire, tick) as in
 * pointid_classify_planes. */
int pointid_gather_planes(const pointid_plane *planes, int32_t n_planes,
                          const int32_t *hits, int64_t n_hits,
                          void *patches_out, int out_dtype, void *stream);

/*
 * One plane binned into columns of D = ticks_per_column ticks (the binning of
 * pointid_classify_planes_ds, alone; needs no handle and runs on the current
 * HIP device).
 *   image  device fp32 [n_wires][n_ticks], any 4-byte alignment
 *   out    device fp32 [n_wires][ceil(n_ticks / D)]: out[w][j] = sum of
 *          image[w][jD + k] over k < D with jD + k < n_ticks, accumulated in
 *          fp64 in tick order and rounded once
 * Errors: EINVAL (n_wires or n_ticks <= 0, ticks_per_column < 1, NULL
 * pointer), EHIP.
 */
int pointid_downsample(const float *image, int32_t n_wires, int32_t n_ticks,
                       int32_t ticks_per_column, float *out, void *stream);

/*
 * Hit finding on deconvolved plane images (paper §2.1: wire hits, with their
 * peak time, are found on the deconvolved waveforms before they are
 * classified; the paper names no algorithm).  Reading used here: tick t of a
 * wire's waveform x is a hit when x[t] > threshold, x[t] > x[t-1] and
 * x[t] >= x[t+1], ticks outside the waveform counting as minus infinity (a
 * plateau gives one hit, at its first tick).  The comparisons are exact fp32
 * comparisons, so the result is bit-exact and deterministic.
 *   planes     HOST array of n_planes descriptors (1 <= n_planes <= 64), read
 *              during the call only; any image alignment
 *   threshold  fp32 (a NaN threshold finds no hit)
 *   hits_out   device int32 [capacity][3] = (plane, wire, tick), in plane, then
 *              wire, then tick order -- the input layout of
 *              pointid_classify_planes; the first min(found, capacity) hits
 *              are written, the rest of the buffer is left as it was
 *   capacity   >= 0; hits_out may be NULL when it is 0
 *   n_found    device int64, 8-byte aligned: receives the number of hits
 *              found, which may exceed capacity (then call again with a larger
 *              buffer); read it after the stream has passed the call
 * Uses the handle's device and scratch cache (about image bytes / 32 of
 * scratch); the network weights are not used.
 * Errors: EINVAL (NULL handle, planes or n_found; misaligned n_found;
 * capacity < 0; NULL hits_out with capacity > 0; a bad plane as in
 * pointid_classify_planes), ENOMEM, EHIP.
 */
int pointid_find_hits(pointid_handle h, const pointid_plane *planes,
                      int32_t n_planes, float threshold, int32_t *hits_out,
                      int64_t capacity, int64_t *n_found, void *stream);

/*
 * Local request server (paper §2.3: the module's model interface sends its
 * inputs to an inference server and blocks until the scores return; many
 * client processes share one GPU and the server merges their requests).
 * pointid_server_start listens on the Unix-domain stream socket
 * `socket_path` (created; it must not exist) and serves each connection on a
 * thread of its own, one request at a time:
 *   - hits (wire, tick) on one of the resident `planes`, or (plane, wire,
 *     tick) over all of them: classified through a dynamic batcher
 *     (pointid_batcher_*, max_requests / max_delay_us) when max_requests > 0,
 *     else by one pointid_classify(_planes) call per request;
 *   - pre-cut fp32 patches (the paper's transmitted inputs):
 *     pointid_classify_patches per request.
 * Scores are bit for bit those of the direct calls.  The handle and the plane
 * images must outlive the server.  A request may hold up to 4,194,304 hits or
 * 65,536 patches; a larger one is refused (EINVAL) and its connection
 * closed.  Wire format: 32-byte request and response headers, then the
 * payload (documented in the library source).
 *   n_planes  0..64 (0: patches only)
 * start errors: EINVAL (NULL handle or out; bad plane; negative sizes; path
 * NULL, empty or longer than 107 bytes), EIO (socket, bind -- e.g. the path
 * exists -- or listen failed), ENOMEM, EHIP.
 * pointid_server_stop closes the socket, lets each connection finish the
 * request it is serving, joins the threads and removes the socket file.
 */
typedef struct pointid_server_s *pointid_server;
int pointid_server_start(pointid_handle h, const pointid_plane *planes,
                         int32_t n_planes, const char *socket_path,
                         int32_t max_requests, int32_t max_delay_us,
                         pointid_server *out);
int pointid_server_stop(pointid_server s);

/*
 * Client of a local request server (plain sockets: no GPU, no HIP call).  All
 * buffers are HOST memory; a call blocks until the scores are back.  One
 * client handle serves one thread at a time.
 *   plane >= 0: hits int32 [n_hits][2] = (wire, tick) on that plane;
 *   plane <  0: hits int32 [n_hits][3] = (plane, wire, tick)
 *   scores fp32 [n][4]
 *   server_ns (optional, may be NULL): time the server spent on the request,
 *   from its header to its scores being ready, in nanoseconds
 * Errors: EINVAL (NULL client or pointer, n_hits out of [0, 4194304] or n
 * patches out of [0, 65536], bad path),
 * EIO (connect, send or receive failed, malformed response), or the status the
 * server returned (EINVAL for a plane it does not hold, ENOMEM, EHIP).
 */
typedef struct pointid_client_s *pointid_client;
int pointid_client_connect(const char *socket_path, pointid_client *out);
int pointid_client_classify(pointid_client c, int32_t plane, const int32_t *hits,
                            int64_t n_hits, float *scores, int64_t *server_ns);
int pointid_client_classify_patches(pointid_client c, const float *patches,
                                    int64_t n, float *scores, int64_t *server_ns);
int pointid_client_close(pointid_client c);

/*
 * Kernel timing for measurement tools (not needed for classification).  While
 * enabled (process-wide), every kernel a classification or hit-finding call
 * launches carries HIP events on its own dispatch (hipExtLaunchKernel), on the
 * stream it runs on (the kernels of pointid_gather[_planes] and
 * pointid_downsample are not timed).  The kernels of one call form a chain:
 * the first is timed from an event recorded on the stream just before it,
 * each later one from the end of the kernel before it, each to its own end
 * (so a kernel's time includes its launch gap, a few microseconds).  Timing
 * adds that one recorded event per call (a gap of about 3.5 us before the
 * first kernel) and turns the call's completion event into a packet of its
 * own (another few microseconds).
 * pointid_timing_query waits for the recorded events of the kernel named
 * `kernel` ("gather", "conv_fc1_16", "conv_fc1_f32", "tail", ...) and returns the
 * summed elapsed milliseconds and the number of launches since the last
 * pointid_timing_reset.  Unknown names return 0 launches.
 * Errors: EINVAL (NULL output pointer), EHIP (event failure).
 */
int pointid_timing_enable(int on);
int pointid_timing_reset(void);
int pointid_timing_query(const char *kernel, double *total_ms, int64_t *launches);

/* Text of the last non-OK status on the calling thread ("" if none). */
const char *pointid_last_error(void);

/* Library version string. */
const char *pointid_version(void);

#ifdef __cplusplus
}
#endif

#endif /* POINTID_H */
