/*
 * trackfit: batched inference of a bidirectional gated linear recurrent
 * encoder that regresses the five perigee parameters (d0, z0, phi, theta, q/p)
 * of a charged-particle track from its time-ordered hit sequence, on AMD
 * Instinct MI355X (gfx950).
 *
 * The method (paper "Fast and Precise Learned Charged-Particle Trajectory
 * Regression at the Large Hadron Collider", Sec. Method and Sec. Encoder):
 * each hit (x, y, z) is min-max normalised and embedded to width d; each of
 * n_layers pre-norm layers applies RMSNorm, one linear projection to a
 * candidate n_t and a gate pre-activation, z_t = sigmoid(gate), the update of
 * Eq. (2) h_t = h_{t-1} + z_t (.) (n_t - h_{t-1}) run forward and in reverse
 * from a zero state, and a linear merge of the two directions added to the
 * residual stream; the stream is averaged over the track's hits and a
 * two-layer head (SiLU between) gives five outputs.
 *
 * C ABI: plain pointers and sizes only.  Device pointers are HIP device
 * memory of the current device; the library never synchronises the stream,
 * never allocates inside fit_tracks, and may therefore be captured in a HIP
 * graph.
 */
#ifndef TRACKFIT_H
#define TRACKFIT_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    TF_OK = 0,
    TF_EINVAL = -1,       /* a host-checkable argument is invalid; nothing was launched */
    TF_ENOMEM = -2,       /* device or host allocation failed (tf_weights_create only) */
    TF_EHIP = -3,         /* a HIP runtime call failed */
    TF_EUNSUPPORTED = -4, /* valid request the library does not implement (e.g. d_model) */
    TF_ETOOLARGE = -5     /* the request exceeds a fixed capacity of the library (nothing was launched) */
} tf_status;

typedef enum { TF_FP32 = 0, TF_BF16 = 1, TF_BF16_F16ACT = 2 } tf_dtype;

/* Model shape and number type.
 * d_model: 32, 64, 128 or 256.  n_layers: 0..64.
 * Projections run on matrix cores with fp32 accumulation in every mode; the
 * gate, both scan states, the residual stream, the mean pool and the outputs
 * are fp32 in every mode (Sec. Kernel adaptation: reduced-precision
 * projections, fp32 recurrence).  The modes differ in the GEMM operands:
 * TF_FP32         fp32 weights and activations.
 * TF_BF16         bf16 weights; the normalised activations and the scan
 *                 outputs are rounded to bf16 as GEMM operands.
 * TF_BF16_F16ACT  weights converted to fp16 operands, activations rounded
 *                 to fp16 (the paper's fp16 projections): same speed as
 *                 TF_BF16 with 3 more mantissa bits on the activations.  A
 *                 bf16 weight converts to fp16 exactly only if its magnitude
 *                 lies in the fp16 normal range [2^-14, 65504]; smaller ones
 *                 lose low bits as fp16 subnormals, larger ones overflow.
 * In both 16-bit modes the RMSNorm gain is folded into the input-projection
 * weights, and the product W_in g is rounded once to the operand type (so it
 * is not the bf16 weight itself), and the two head layers multiply their fp32
 * input as a high and a low 16-bit part. */
typedef struct {
    int32_t n_layers;
    int32_t d_model;
    int32_t dtype;    /* tf_dtype */
    int32_t max_hits; /* longest track the caller will pass; 0 = the largest
                         supported (64 for d_model <= 128, 32 for 256).  Up to
                         32 selects the one-tile-per-wave kernel, which is
                         faster; longer tracks then get NaN and an error flag. */
    int32_t n_features; /* 0: hits are (x, y, z) and the model embeds them
                           linearly.  1..16: the paper's front end (Sec.
                           Encoder): hits carry n_features values per hit, each
                           min-max normalised, u = (x - lo) * (1 / (hi - lo))
                           with every step rounded to float32, expanded to
                           sin(pi 2^s u) and cos(pi 2^s u) for s = 0..15, and
                           the 32 n_features values projected linearly to
                           d_model.  Supported for d_model 32 and 128. */
} tf_config;

/* Opaque: device-resident weights in kernel order plus a sticky device error
 * word.  Owned by the library. */
typedef struct tf_weights tf_weights;

/*
 * Copy a canonical float32 weight blob to the current device: the parameters
 * of the encoder that fit_tracks evaluates (Sec. Encoder, Eq. (2) per layer).
 *
 * Blob order (matrices row-major [out][in]):
 *   embed.W[d][3], embed.b[d],
 *   per layer: norm.g[d], in.W[3d][d], in.b[3d], out.W[d][2d], out.b[d],
 *   head.W1[d][d], head.b1[d], head.W2[5][d], head.b2[5].
 * Rows 0..d-1 of in.W give the candidate, rows d..2d-1 the gate
 * pre-activation, rows 2d..3d-1 are unused.  Columns 0..d-1 of out.W read the
 * forward state, d..2d-1 the reverse state.  n_floats must equal
 * tf_blob_size(n_layers, d_model) (tf_fourier_blob_size with a Fourier front
 * end).  In the 16-bit modes the matrix values should already be
 * bf16-representable; others are rounded to nearest even.
 *
 * Ownership: host_blob is only read during the call.  *out receives a handle
 * the caller frees with tf_weights_destroy.  Synchronous.
 * Errors: TF_EINVAL (null pointers, bad sizes, max_hits < 0, n_features < 0),
 * TF_EUNSUPPORTED (d_model, n_layers, max_hits or n_features outside the
 * supported set),
 * TF_ENOMEM, TF_EHIP.  On error *out is set to NULL.
 */
tf_status tf_weights_create(const tf_config *cfg, const float *host_blob, size_t n_floats,
                            tf_weights **out);

/* Free a handle (NULL is a no-op).  Synchronises the device first. */
void tf_weights_destroy(tf_weights *w);

/* Number of floats of the canonical blob for a model shape (0 if invalid). */
size_t tf_blob_size(int32_t n_layers, int32_t d_model);

/* Number of floats of the blob of a model with the Fourier front end over
 * n_features (1..16) per-hit features, 0 if invalid.  Its order replaces
 * embed.W and embed.b of the canonical blob by
 *   fe.lo[F], fe.hi[F], fe.W[d][32 F], fe.b[d]
 * where column 32 f + 16 c + s of fe.W reads sin (c = 0) or cos (c = 1) of
 * pi 2^s u_f, the normalised feature f at scale s. */
size_t tf_fourier_blob_size(int32_t n_layers, int32_t d_model, int32_t n_features);

/* Longest track (in hits) the kernels accept for this handle: 32 or 64, from
 * tf_config.max_hits.  Longer tracks get NaN outputs and set
 * TF_DEVERR_TOO_LONG. */
int32_t tf_max_hits(const tf_weights *w);

/*
 * Fit a packed batch of tracks (Sec. Kernel adaptation: packed, unpadded
 * layout; the problem statement of Sec. Method: one ordered hit sequence in,
 * five perigee parameters out).
 *
 * hits     device, float32 [n_hits][3] = (x, y, z) in mm, time-ordered within
 *          each track; with the Fourier front end [n_hits][n_features], the
 *          per-hit features in the order of fe.lo / fe.hi.  Read only.
 * n_hits   rows of hits (bounds every read: a track whose rows leave
 *          [0, n_hits) gets NaN outputs and sets TF_DEVERR_BAD_OFFSETS).
 * offsets  device, int32 [n_tracks + 1]: track i owns rows
 *          offsets[i] .. offsets[i+1]-1.  Non-decreasing; offsets[0] may be > 0
 *          (absolute offsets into a larger array).  Read only.
 * n_tracks host scalar >= 0.  0 is a no-op returning TF_OK.
 * w        weights from tf_weights_create (same device).
 * out      device, float32 [n_tracks][5]: d0, z0, phi, theta, q/p order.
 *          Every row is written.  Must not overlap the inputs.
 * stream   HIP stream (0 = null stream).
 *
 * Asynchronous: returns after enqueueing; no allocation, no host sync, so the
 * call can be captured into a HIP graph.  Tracks with zero hits, more than
 * tf_max_hits hits, a decreasing offset or rows outside [0, n_hits) get NaN
 * outputs and set the sticky device error word (tf_get_device_error).
 * A handle may be used from several streams at once.
 * Errors: TF_EINVAL (null pointers with n_tracks > 0, n_tracks < 0,
 * n_hits < 0), TF_EHIP (launch failure).
 */
tf_status fit_tracks(const float *hits, int64_t n_hits, const int32_t *offsets, int32_t n_tracks,
                     const tf_weights *w, float *out, hipStream_t stream);

/*
 * The paper's readout input instead of the pooled head (Sec. Encoder, last
 * paragraph: the forward state at the outermost hit and the reverse state at
 * the innermost hit of the last layer, concatenated).  Runs the same encoder
 * as fit_tracks and stops after the last layer's scans: that layer's output
 * projection and the pooled head are not evaluated.
 *
 * states   device, float32 [n_tracks][2 d]: columns 0 .. d-1 hold the last
 *          layer's forward scan state at the track's last hit, columns
 *          d .. 2d-1 its reverse scan state at the track's first hit (both
 *          before the output projection).  Every row is written; rejected
 *          tracks (as for fit_tracks) get NaN rows.  Must not overlap the
 *          inputs.
 * Other arguments, asynchrony and device errors as for fit_tracks.
 * Errors: as fit_tracks, and TF_EUNSUPPORTED for a model with no layers.
 */
tf_status fit_tracks_states(const float *hits, int64_t n_hits, const int32_t *offsets, int32_t n_tracks,
                            const tf_weights *w, float *states, hipStream_t stream);

/* Bits of the sticky device error word. */
#define TF_DEVERR_EMPTY_TRACK 1   /* a track with zero hits */
#define TF_DEVERR_TOO_LONG 2      /* a track longer than tf_max_hits */
#define TF_DEVERR_BAD_OFFSETS 4   /* decreasing offsets or rows outside [0, n_hits) */
#define TF_DEVERR_PAIR 8          /* internal: in a 64-hit launch, a wave gave up waiting for the
                                     other wave of its tile (the launch's outputs are not valid) */

/* Read (and if clear != 0, reset) the sticky device error word after the work
 * already enqueued on stream.  Synchronises stream.  *flags receives the OR of
 * TF_DEVERR_* bits seen since the last clear.  (Library plumbing: no passage of
 * the paper defines it; it reports the tracks the kernels refused.) */
tf_status tf_get_device_error(const tf_weights *w, hipStream_t stream, int32_t *flags, int clear);

/*
 * Analytic three-hit seed of every track, and optionally the per-hit seed
 * residual features (Sec. Method, "Analytic seed"; fp64 throughout, as the
 * paper computes the seed).
 *
 * Seed: the circle through the track's first three hits in the transverse
 * plane gives pT = 0.299792458 * b_tesla * R[m] and the charge (field along
 * +z: a positive track turns clockwise seen from +z), its closest approach to
 * the z axis the perigee (d0, phi), and the transverse arc lengths of the
 * first and third hit from the perigee give theta and z0.  Conventions: the
 * perigee point is d0 * (-sin phi, cos phi) and phi the direction of motion
 * there; theta in (0, pi); q/p in 1/GeV.
 * Features of each hit: asinh(dU), asinh(dV) and the helix path length from
 * the perigee (mm), where (dU, dV) is the hit's residual to the seed helix in
 * the curvilinear frame of the helix (dU transverse, dV along the other
 * direction normal to the motion), in mm.
 *
 * hits      device, float32 [n_hits][3] = (x, y, z) in mm, time-ordered within
 *           each track (the first three hits make the seed).  Read only.
 * n_hits    rows of hits (bounds every read).
 * offsets   device, int32 [n_tracks + 1], as for fit_tracks.  Read only.
 * n_tracks  host scalar >= 0.  0 is a no-op returning TF_OK.
 * b_tesla   host scalar > 0: solenoid field along +z.
 * seeds     device, float64 [n_tracks][5]: d0 [mm], z0 [mm], phi, theta,
 *           q/p [1/GeV].  Every row is written.
 * features  device, float32 rows of feature_stride floats, or NULL to skip
 *           them: the three features of hit row offsets[0] + r are at
 *           features[r * feature_stride + 0 .. 2], for r < offsets[n_tracks] -
 *           offsets[0] (with feature_stride = 15 and features pointing at
 *           column 12, the seed fills the last three columns of the Fourier
 *           front end's per-hit feature rows).
 * feature_stride  host scalar: 0 or 3 for packed rows, else >= 3.
 * flags     device int32 or NULL: OR-ed with TF_SEED_* bits of the tracks that
 *           got NaN seeds (their features are NaN too, unless their offsets
 *           are bad, in which case their rows are not written).
 * stream    HIP stream (0 = null stream).
 *
 * Asynchronous, allocates nothing (graph-capturable).  Outputs must not
 * overlap the inputs.  Errors: TF_EINVAL (null pointers with n_tracks > 0,
 * negative sizes, b_tesla <= 0, feature_stride 1 or 2 or negative), TF_EHIP
 * (launch failure).
 */
tf_status tf_seed_tracks(const float *hits, int64_t n_hits, const int32_t *offsets, int32_t n_tracks,
                         double b_tesla, double *seeds, float *features, int32_t feature_stride, int32_t *flags,
                         hipStream_t stream);

/* Bits of tf_seed_tracks' flags. */
#define TF_SEED_TOO_SHORT 1    /* fewer than three hits */
#define TF_SEED_NO_CIRCLE 2    /* two of the first three hits coincide in the transverse plane, or the
                                  three are collinear */
#define TF_SEED_BAD_OFFSETS 4  /* decreasing offsets, or rows outside [0, n_hits) or outside
                                  [offsets[0], offsets[n_tracks]) */

/*
 * The paper's readout and decode (Sec. Encoder, last paragraph: RMSNorm of the
 * end states and a two-layer head of hidden width 128 with 35 outputs; Sec.
 * Losses: seven quantiles per parameter, the median quantile as the point
 * estimate; Sec. Method: the prediction is a correction to the analytic
 * seed).  The head's activation is SiLU.
 *
 * Opaque: the head's weights in kernel order on the device.  Owned by the
 * library.
 */
typedef struct tf_readout tf_readout;

/* Number of floats of a readout head blob for end states of width 2d and a
 * hidden layer of `hidden` units (0 if invalid):
 * norm.g[2d], W1[hidden][2d], b1[hidden], W2[35][hidden], b2[35]
 * (row-major [out][in]).  Output 7 p + i of W2 is quantile i of parameter p
 * (d0, z0, phi, theta, q/p order), the quantiles in increasing order of their
 * levels, so that output 7 p + 3 is the median quantile (level 1/2). */
size_t tf_readout_blob_size(int32_t d, int32_t hidden);

/* Copy a readout head blob to the current device.  d: a multiple of 32 up to
 * 256 (192 for the paper's backbone: states of 2 x 192); hidden: a multiple
 * of 32 up to 256 (the paper's head: 128).
 * dtype (tf_dtype): TF_FP32 runs the head's products in fp32; TF_BF16 and
 * TF_BF16_F16ACT (the 16-bit models) take W1 and W2 in bf16 (exact for
 * bf16-valued weights; others are rounded to nearest even) and multiply them
 * with the fp32 activations (the gain applied in fp32) split into a high and
 * a low bf16 part (about 16 significant bits), accumulating in fp32.
 * host_blob is only read during the call; *out receives a handle freed with
 * tf_readout_destroy.  Synchronous; allocates device memory.
 * Errors: TF_EINVAL (null pointers, n_floats != tf_readout_blob_size(d,
 * hidden), unknown dtype), TF_EUNSUPPORTED (other d or hidden), TF_ENOMEM,
 * TF_EHIP.  On error *out is NULL. */
tf_status tf_readout_create(int32_t d, int32_t hidden, int32_t dtype, const float *host_blob, size_t n_floats,
                            tf_readout **out);

/* Free a handle (NULL is a no-op).  Synchronises the device first. */
void tf_readout_destroy(tf_readout *h);

/*
 * Readout, point estimates and decode of a batch of tracks:
 *   y = g (.) z / sqrt(mean(z^2) + 1e-6),  h = SiLU(W1 y + b1),
 *   q = W2 h + b2,  m_p = q[7p + 3] (parameter p's median quantile),
 *   d0, z0, theta: seed + m;  phi: seed + m wrapped to [-pi, pi);
 *   q/p: seed + m * (|seed| + 0.02 / GeV).
 * The head runs on matrix cores with fp32 accumulation in the handle's number
 * type; the decode in fp64.
 *
 * states    device, float32 [n_tracks][2d], as written by fit_tracks_states
 *           (d of the handle).  Read only.
 * n_tracks  host scalar >= 0.  0 is a no-op returning TF_OK.
 * seeds     device, float64 [n_tracks][5], as written by tf_seed_tracks.
 * h         handle from tf_readout_create (same device).
 * quantiles device, float32 [n_tracks][35] or NULL to skip them: q per track.
 * out       device, float64 [n_tracks][5]: the decoded d0 [mm], z0 [mm], phi,
 *           theta, q/p [1/GeV].  Every row is written.  A track whose states
 *           or seed hold a NaN gets NaN in the affected outputs.
 * stream    HIP stream (0 = null stream).
 *
 * Asynchronous, allocates nothing (graph-capturable).  Outputs must not
 * overlap the inputs.  Errors: TF_EINVAL (null pointers with n_tracks > 0,
 * n_tracks < 0), TF_EHIP (launch failure).
 */
tf_status tf_decode_tracks(const float *states, int32_t n_tracks, const double *seeds, const tf_readout *h,
                           float *quantiles, double *out, hipStream_t stream);

/*
 * The paper's own backbone (Sec. Encoder, Eq. (2)): a stack of bidirectional
 * minGRU layers of H channels per direction behind the front end.  Per layer,
 * four linear maps of the input give the forward and the reverse pass a
 * candidate and a gate each (z = sigmoid(gate)); the passes run the update of
 * Eq. (2) from each track's first hit and from its last (zero initial state),
 * and [f; b] (2H values per hit) feeds the next layer; no normalisation or
 * residual inside.
 * Number types as for tf_config.dtype: fp32 throughout, or 16-bit matrix
 * operands (weights bf16, activations bf16 or fp16) with fp32 accumulation,
 * gates and recurrence.
 */
typedef struct {
    int32_t n_layers;   /* 1..8 */
    int32_t d_model;    /* front-end width: 32 (with H = 64) or 128 (with H = 192) */
    int32_t hidden;     /* H */
    int32_t dtype;      /* tf_dtype */
    int32_t n_features; /* 0: (x, y, z) front end; 1..16: the Fourier front end */
} tf_mingru_config;

typedef struct tf_mingru tf_mingru;

/* Floats of the blob (0 if invalid).  Order (float32, row-major [out][in]):
 * the front end as in tf_weights_create's blob (embed.W[d][3], embed.b[d], or
 * fe.lo[F], fe.hi[F], fe.W[d][32 F], fe.b[d]), then per layer l: W[4H][D_l],
 * b[4H] with D_0 = d and D_l = 2H; rows 0..H-1 forward candidate, H..2H-1
 * forward gate pre-activation, 2H..3H-1 reverse candidate, 3H..4H-1 reverse
 * gate pre-activation; columns of a later layer read [f; b] of the one
 * before (forward state first). */
size_t tf_mingru_blob_size(const tf_mingru_config *cfg);

/* Copy a blob to the current device.  Synchronous; allocates device memory.
 * Tracks may have up to 32 hits.  Errors: TF_EINVAL (null pointers, bad
 * sizes or dtype), TF_EUNSUPPORTED (other widths, more than 8 layers, more
 * than 16 features), TF_ENOMEM, TF_EHIP.  On error *out is NULL. */
tf_status tf_mingru_create(const tf_mingru_config *cfg, const float *host_blob, size_t n_floats, tf_mingru **out);

/* Free a handle (NULL is a no-op).  Synchronises the device first. */
void tf_mingru_destroy(tf_mingru *h);

/* Bytes of device workspace tf_mingru_states needs for a batch of n_rows hit
 * rows (offsets[n_tracks] - offsets[0]): the front end's output and up to two
 * layer outputs, row-major, in the operand type. */
size_t tf_mingru_workspace_size(const tf_mingru *h, int64_t n_rows);

/*
 * End states of the last layer for a packed batch: the readout's input
 * (Sec. Encoder, last paragraph).
 *
 * hits, n_hits, offsets, n_tracks  as for fit_tracks (hits carry n_features
 *           values per hit with the Fourier front end).
 * workspace device memory of workspace_bytes (see tf_mingru_workspace_size);
 *           its contents are scratch.  Tracks whose rows do not fit get NaN.
 * states    device, float32 [n_tracks][2H]: the forward state at the track's
 *           last hit, then the reverse state at its first hit.  Every row is
 *           written; tracks with no hits, more than 32 hits or rows outside
 *           [0, n_hits) get NaN rows and set the device error word.
 * Asynchronous, allocates nothing.  One launch for the front end, one per
 * layer, all on stream; or, for the paper's deployed configuration (16-bit
 * modes, Fourier front end, d_model 128, hidden 192, two layers) and unless
 * tf_mingru_set_fused turned it off, one fused launch that keeps the front
 * end's output and the first layer's states on chip (same results, bit for
 * bit; the workspace is then left untouched but still bounds the rows).
 * Errors: TF_EINVAL (null pointers with n_tracks > 0, negative sizes),
 * TF_EHIP (launch failure).
 */
tf_status tf_mingru_states(const float *hits, int64_t n_hits, const int32_t *offsets, int32_t n_tracks,
                           const tf_mingru *h, void *workspace, size_t workspace_bytes, float *states,
                           hipStream_t stream);

/*
 * Choose how tf_mingru_states and tf_mingru_states_noalloc run the paper's
 * deployed configuration (Sec. Kernel adaptation: the front end and the token
 * mixing of the layers fused on chip): fused != 0 one launch (the default
 * where it applies), 0 the layered launches.  Not to be called while calls
 * on the handle are in flight.  Errors: TF_EINVAL (NULL handle),
 * TF_EUNSUPPORTED (fused asked for another configuration; the handle keeps
 * the layered path).
 */
tf_status tf_mingru_set_fused(tf_mingru *h, int fused);

/*
 * tf_mingru_states for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same kernels and results, with the workspace taken from a fixed
 * 128 MiB array that the library keeps in device memory, one copy per device,
 * for the life of the process (looked up once per device in tf_mingru_create,
 * on the device current there).  The call itself allocates nothing and
 * never synchronises.
 *
 * Arguments as for tf_mingru_states, without the workspace.  The hit array
 * may have at most tf_mingru_noalloc_max_rows(h) rows (n_hits): offsets then
 * index it from row 0 up, so every row of the batch fits.
 * All calls on one device share that device's array and leave their rows in
 * it; nothing needs clearing between calls (every row a kernel reads was
 * written earlier in the same call).  Calls that overlap in time on one
 * device (other streams, other handles, other threads) race on the array and
 * must be ordered by the caller.
 * Errors: TF_EINVAL (as tf_mingru_states), TF_ETOOLARGE (n_hits above
 * tf_mingru_noalloc_max_rows(h); nothing launched), TF_EHIP.
 */
tf_status tf_mingru_states_noalloc(const float *hits, int64_t n_hits, const int32_t *offsets, int32_t n_tracks,
                                   const tf_mingru *h, float *states, hipStream_t stream);

/* Rows of hits tf_mingru_states_noalloc accepts for this handle (0 for NULL):
 * 128 MiB over the workspace bytes per row (1 KiB per row for d_model 128,
 * H 192, two layers, 16-bit operands: 131071 rows). */
int64_t tf_mingru_noalloc_max_rows(const tf_mingru *h);

/* Read (and if clear != 0, reset) the handle's sticky device error word
 * (TF_DEVERR_* bits).  Synchronises stream. */
tf_status tf_mingru_device_error(const tf_mingru *h, hipStream_t stream, int32_t *flags, int clear);

/* Static description of a status code (library plumbing: no passage of the
 * paper defines it). */
const char *tf_status_string(tf_status s);

#ifdef __cplusplus
}
#endif

#endif /* TRACKFIT_H */
