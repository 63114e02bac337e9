/*
 * sketch.h -- C ABI of the MI355X (gfx950) structured-sketch library.
 *
 * A sketch is a seeded random linear map S: R^N -> R^D applied to a batch of
 * vectors that arrive as a ragged list of parameter tensors ("layers"), and its
 * transpose S^T: R^D -> R^N.  Kinds, following "Efficient Sketches for
 * Training Data Attribution and Studying the Loss Landscape" (Schioppa,
 * NeurIPS 2024):
 *
 *   SK_FJL   y = sqrt(N/D) G_s H_N B x                  (eq. ailon_chazelle)
 *   SK_FFD   y = sum_b B_b H_D Pi_b^T G_b H_D x_b         (eq. fastfood, used as
 *            the transpose of the feature map; sigma_F = 1 as in the proof of
 *            Thm. fastfood_bad_inputs)
 *   SK_AFFD  y = R_D(sqrt(N/D) H^{pi2}_N G H^{pi1}_N B x) (eq. bami)
 *   SK_AFJL  y = R_D(sqrt(N/D) G H^{pi1}_N B x)           (eq. frikadel)
 *   SK_QK    Y = A X B^T per weight matrix X (m x n), A (dA x m) ~ N(0,1/dA),
 *            B (dB x n) ~ N(0,1/dB)                       (eq. straight with two
 *            Kronecker factors, contraction of eq. qk_proof_tensor_dec)
 *   SK_QKH   y = sqrt(N/D) R_D Q_N x                      (eq. straight on the
 *            flattened layer: Q_N is the Kronecker product of Haar-orthogonal
 *            factors of the sizes of N, restricted to their first D_i rows)
 *   SK_AFJLQ y = sqrt(N/D) G R_D Q_N x                    (eq. frikadel with the
 *            pre-conditioner H_N replaced by Q, Sec. 3 "Alternative
 *            pre-conditioners")
 *   SK_AFFDQ y = sqrt(N/D) R_D Q'_N G Q_N x               (eq. bami with both
 *            H_N replaced by independent Q_N, Q'_N; G over N'.  Dense work:
 *            about 4 GFLOP per vector and 2^20-element slab)
 *   SK_AFJLF y = sqrt(N/D) G R_D F_N B x                  (eq. frikadel with the
 *            pre-conditioner H_N replaced by the FFT, Sec. 3 "Alternative
 *            pre-conditioners".  F_N is the real orthonormal Fourier matrix:
 *            rows 1/sqrt(N), (-1)^n/sqrt(N), then per frequency k >= 1 the
 *            pair sqrt(2/N) (cos, -sin)(2 pi k n / N); so y holds X_0, X_{N/2}
 *            and Re, Im of X_1 .. X_{D/2-1} of the DFT X of B x, scaled)
 *
 * H_N is the normalised Walsh-Hadamard matrix (appendix definition), R_D keeps
 * the first D coordinates, B is a diagonal of random signs, G a diagonal of
 * N(0,1) entries, and pi1/pi2 permute digits within the Kronecker factors of N
 * (Sec. 3, "Removing the lookup bottleneck"; factors of at most 1024).
 *
 * Per layer l with n_l = rows*cols elements the FWHT kinds (and SK_QKH,
 * SK_AFJLQ, SK_AFFDQ) work on the padded length N'_l = 2^ceil(log2 max(n_l, D)) (padding
 * is virtual: never read or written).  They sum independent per-layer sketches
 * (each with its own random streams, keyed on the layer's index in the list),
 * which is the
 * per-shard lift followed by a sum of the paper's model-parallel appendix.  QK
 * concatenates the dA*dB blocks of its layers in list order (sum dA*dB = D).
 *
 * Every random quantity is regenerated from (seed, layer, stream, index) with a
 * counter-based Philox4x32-10 generator; nothing of size N is stored.
 *
 * Conventions for every entry point:
 *  - Return 0 (SK_OK) on success, a negative SK_E* code on failure.  Arguments
 *    are validated before any device work is queued; on failure no output
 *    buffer is touched.  sketch_last_error() gives a thread-local message.
 *  - Device pointers are plain HIP device addresses on the sketch's device;
 *    the arrays OF pointers (grads, out, theta0) are host memory and are read
 *    during the call only.
 *  - Work is queued asynchronously on `stream` (a hipStream_t; NULL = the
 *    legacy default stream).  Results are ready when the stream is.
 *  - A handle is immutable after creation, but owns one workspace: calls on the
 *    same handle must be serialised on one stream (not thread-safe).
 *  - The caller owns all input/output buffers; the handle owns its tables and
 *    workspace, allocated at creation.  Apply calls never allocate or free.
 *  - Results are bitwise deterministic for a fixed build, device, sketch and
 *    input (no floating-point atomics).
 */
#ifndef SK_SKETCH_H
#define SK_SKETCH_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SK_FJL = 0,
  SK_FFD = 1,
  SK_AFFD = 2,
  SK_AFJL = 3,
  SK_QK = 4,
  SK_QKH = 5,
  SK_AFJLQ = 6,
  SK_AFFDQ = 7,
  SK_AFJLF = 8
} sk_kind;
typedef enum { SK_F32 = 0, SK_BF16 = 1 } sk_dtype;

enum {
  SK_OK = 0,
  SK_EINVAL = -1,      /* bad argument: kind, D, shapes, null pointer, batch  */
  SK_EDTYPE = -2,      /* unknown dtype                                       */
  SK_ENOMEM = -3,      /* device allocation failed at creation                */
  SK_EHIP = -4,        /* a HIP runtime call failed                           */
  SK_EUNSUPPORTED = -5 /* valid in the math but outside what the kernels take */
};

/* One parameter tensor, row-major rows x cols (1-D tensors: rows = 1).
 * qk_da, qk_db: the QK output block shape of this matrix (1 <= qk_da <= rows,
 * 1 <= qk_db <= cols); ignored by the other kinds. */
typedef struct {
  int64_t rows, cols;
  int32_t qk_da, qk_db;
} sk_layer_shape;

typedef struct sk_sketch sk_sketch;

/* Introspection record (sketch_query). */
typedef struct {
  int32_t kind, n_layers;
  int64_t D;
  uint64_t seed;
  int64_t total_numel;      /* sum of rows*cols                      */
  int64_t total_padded;     /* sum of N'_l (FWHT kinds), else 0      */
  int64_t workspace_bytes;  /* device workspace owned by the handle  */
  int32_t rng_version;      /* version of the random-stream layout   */
  int32_t device;
} sk_info;

/* Random-stream identifiers (the fourth Philox counter word). */
enum {
  SK_STREAM_SIGN = 1,    /* B signs, one per coordinate of N'_l            */
  SK_STREAM_GAUSS = 2,   /* G entries (AFFD, FFD: N'_l; FJL, AFJL, AFJLF: D) */
  SK_STREAM_INDEX = 3,   /* FJL sample positions in [0, N'_l)              */
  SK_STREAM_FFDPERM = 4, /* FFD block permutation Pi_b                     */
  SK_STREAM_PI1 = 5,     /* digit permutation before the first H           */
  SK_STREAM_PI2 = 6,     /* digit permutation after the second H (AFFD)    */
  SK_STREAM_QKA = 7,     /* QK left factor                                 */
  SK_STREAM_QKB = 8,     /* QK right factor                                */
  SK_STREAM_QH = 9       /* SK_QKH / SK_AFJLQ / SK_AFFDQ factor k of a layer
                            (SK_AFFDQ second set: k = 8 + digit): Gaussian
                            numbers k 2^20 + r b + c form the b x b matrix
                            whose normalised QR factor (R with a positive
                            diagonal) is factor k; computed in fp64 on the
                            host at creation, stored in fp32               */
};

/*
 * Create a sketch on HIP device `device`.
 *   kind      one of sk_kind.
 *   shapes    host array of n_layers >= 1 layer shapes (rows, cols >= 1).
 *   D         target dimension.  FWHT kinds: a power of two, 16 <= D <= 2^20
 *             (D > 2^20 is SK_EUNSUPPORTED).  QK: D = sum qk_da*qk_db.
 *             SK_QKH, SK_AFJLQ, SK_AFFDQ: a power of two, 2048 <= D <= 2^20
 *             (smaller D is SK_EUNSUPPORTED by the kernels); SK_AFFDQ also
 *             needs N'_l <= 2^26 for every layer.  SK_FJL needs N'_l <= 2^32
 *             (a sample position is one 32-bit random word masked to N'_l - 1;
 *             larger layers are SK_EUNSUPPORTED).  SK_AFJLF: a power of two,
 *             2048 <= D <= 2^20; a layer with N'_l = D needs at most 16384
 *             entries or D <= 2^16, and layers with D < N'_l < 128 D need
 *             D^2/(4 N'_l) <= 16384 (D >= 2^17 excludes some; otherwise
 *             SK_EUNSUPPORTED).
 *             Every layer: rows*cols <= 2^40.
 *   seed      64-bit key of every random stream.
 *   flags     0 or SK_FLAG_AFFD_NO_MTAB (see below).
 * On success *out receives the handle (destroy with sketch_destroy).  The
 * small per-layer tables and the QK factors are generated on the device here
 * (QK: A in fp32; B in fp32 split into two bf16 terms for the MFMA units).
 */
int sketch_create(sk_kind kind, const sk_layer_shape *shapes, int32_t n_layers, int64_t D, uint64_t seed,
                  uint32_t flags, int32_t device, sk_sketch **out);

/*
 * AFFD layers whose second-to-last Kronecker digit has 1024 values: by default
 * sketch_create stores, per such layer, the N'_l values
 *   M[t'][p][l] = sum_t H[t][t'] (-1)^<h*, t> g[t, p, l]
 * (the Gaussian diagonal G combined with the signed top-digit fold; fp32, one
 * copy per sketch) when all of them together fit in SK_AFFD_MTAB_MB MiB of
 * device memory (environment, default 8192), so that sketch_apply reads them
 * instead of regenerating G.  With SK_FLAG_AFFD_NO_MTAB nothing is stored and
 * G is regenerated on every call; the results agree to rounding.
 */
#define SK_FLAG_AFFD_NO_MTAB 1u

/*
 * FFD with D = 2^20: for every live block, sketch_create stores where each
 * group of 8 source columns starts its run inside the bucket of each run of
 * 8 destination rows, for Pi_b and its inverse (uint16, 64 KB per block), when
 * all of them fit in SK_FFD_BUCKET_MB MiB (environment, default 1024).  Calls
 * on batches that are a multiple of 4 then permute through those buckets;
 * without the tables they gather through Pi_b.  The results are identical.
 */

/*
 * Forward sketch y = sum over the selected layers of S_l x_l.
 *   grads       host array of n_layers device pointers; grads[i] holds layer
 *               first_layer+i as [batch, rows*cols] row-major, contiguous, in
 *               `dtype` (SK_F32 or SK_BF16 bit patterns), 4-byte aligned.
 *   batch       number of vectors (0 is a no-op).
 *   out         device [batch, D] fp32.  accumulate = 0 overwrites, 1 adds to
 *               what `out` holds (streaming a model layer group by layer
 *               group).  For QK only the selected layers' column blocks of
 *               `out` are written (or accumulated).
 *   first_layer, n_layers  the contiguous layer range this call covers.
 * Arithmetic is fp32 (bf16 inputs are widened exactly); QK multiplies bf16
 * inputs by the bf16 hi and lo terms of B on the matrix cores with fp32
 * accumulation, then by the fp32 A.
 */
int sketch_apply(sk_sketch *s, const void *const *grads, sk_dtype dtype, int64_t batch, float *out,
                 int32_t first_layer, int32_t n_layers, int32_t accumulate, void *stream);

/*
 * sketch_apply without any allocation or use of the handle's workspace, for
 * callers that cannot allocate device memory: code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc.  Arguments, results
 * and errors are those of sketch_apply.  The per-call scratch is a static
 * device array of 64 MiB (SK_STATIC_SCRATCH_BYTES) that each device the
 * library runs on holds until the process ends; its device address is looked
 * up on the first call on each device (hipGetSymbolAddress, which may fail with
 * SK_EHIP).  Layer ranges whose one vector needs more scratch than that (for
 * instance AFFD or FJL layers of 2^24 or more padded elements, AFJL with
 * D = 2^20, QK matrices whose first stage holds more than 16 M floats per
 * vector) are rejected with SK_EUNSUPPORTED before any launch, leaving `out`
 * untouched; larger batches go through in chunks that fit.  The kernels write
 * every scratch element they read, so leftovers of earlier calls do not
 * matter.  All calls on one device share its array: calls that may overlap in
 * time on one device (other streams, other host threads, other handles) race
 * and must be serialised by the caller.
 */
#define SK_STATIC_SCRATCH_BYTES (64ll << 20)
int sketch_apply_noalloc(sk_sketch *s, const void *const *grads, sk_dtype dtype, int64_t batch, float *out,
                         int32_t first_layer, int32_t n_layers, int32_t accumulate, void *stream);

/*
 * Transpose x_l = S_l^T z (+ theta0_l) for the selected layers.
 *   z        device [batch, D] fp32.
 *   out      host array of n_layers device pointers, out[i] is
 *            [batch, rows*cols] of layer first_layer+i in `out_dtype`
 *            (bf16 outputs are rounded to nearest even).
 *   theta0   NULL, or a host array of n_layers device pointers, each NULL or
 *            an fp32 [rows*cols] vector broadcast-added over the batch (the
 *            intrinsic-dimension reparameterisation theta0 + S^T z).
 */
int sketch_apply_T(sk_sketch *s, const float *z, int64_t batch, void *const *out, sk_dtype out_dtype,
                   const void *const *theta0, int32_t first_layer, int32_t n_layers, void *stream);

/* Free everything the handle owns (synchronises its device).  NULL is a no-op. */
void sketch_destroy(sk_sketch *s);

/* Fill *info.  Returns SK_EINVAL on NULL arguments. */
int sketch_query(const sk_sketch *s, sk_info *info);

/*
 * Regenerate `count` values of a random stream ON THE DEVICE, starting at
 * index `start`, and copy them to host memory `host_out` (synchronous).
 *   SK_STREAM_SIGN               int8 +-1 per coordinate.
 *   SK_STREAM_GAUSS/QKA/QKB      fp32 N(0,1) values (QK factors before the
 *                                1/sqrt(d) scale and bf16 rounding).
 *   SK_STREAM_INDEX              uint32 positions in [0, N'_layer).
 *   SK_STREAM_PI1/PI2            uint32 pi(i) of the full digit permutation
 *                                of [0, N'_layer).
 *   SK_STREAM_FFDPERM            uint32 pi_b(i) on [0, D), b = `aux`.
 * Out-of-range indices give SK_EINVAL.
 */
int sketch_debug_stream(sk_sketch *s, int32_t layer, int32_t stream_id, uint64_t start, uint64_t count,
                        uint64_t aux, void *host_out);

/*
 * Kernel timing (diagnostics and roofline reports).  While profiling is on,
 * every group of kernel launches of a selected class that a call issues is
 * bracketed by HIP events on that call's stream, tagged with the class and the
 * algorithmic bytes the group moves (inputs read once plus outputs written
 * once).  sketch_profile(s, classes) with a nonzero bit mask (bit c selects
 * class c below; SK_PROF_ALL selects every class) allocates the event pool (up
 * to 16384 groups) on first use and clears the record; sketch_profile(s, 0)
 * stops recording; bits outside SK_PROF_ALL give SK_EINVAL.  Each event pair
 * costs a little device time, so selecting only the class of interest keeps
 * the timed stream closest to an unprofiled one.  sketch_profile_read()
 * waits for the recorded events and fills, per class (arrays of
 * SK_PROF_CLASSES entries), the summed duration in ms, the number of groups
 * and the summed algorithmic bytes, then clears the record.
 */
enum {
  SK_PROF_AFJL_FOLD = 0, /* AFJL row fold + H_L                           */
  SK_PROF_AFJL_TAIL = 1, /* AFJL H_R, G, layer sum                          */
  SK_PROF_FWHT = 2,      /* generic Walsh-Hadamard passes                   */
  SK_PROF_PROLOG = 3,    /* load / sign / permute of inputs (AFFD, FJL)     */
  SK_PROF_AFFD_FOLD = 4, /* AFFD G + signed fold of the top digits          */
  SK_PROF_GATHER = 5,    /* final gathers and output writes                 */
  SK_PROF_FFD = 6,       /* FFD block kernels                               */
  SK_PROF_QK = 7,        /* QK contractions                                 */
  SK_PROF_OTHER = 8,
  SK_PROF_AFFD_ROWS = 9, /* AFFD row kernel: load, sign, pi1, H_l (one launch) */
  SK_PROF_QK_XB = 10,    /* QK first contraction X B^T (reads the gradients) */
  SK_PROF_QH_FIRST = 11, /* SK_QKH/SK_AFJLQ contraction that reads the input */
  SK_PROF_QH_SECOND = 12,/* SK_QKH/SK_AFJLQ/SK_AFFDQ second contraction        */
  SK_PROF_QH_T = 13,     /* SK_QKH/SK_AFJLQ/SK_AFFDQ transposes               */
  SK_PROF_FFD_T = 14,    /* FFD transpose with D <= 2^13 (one launch)        */
  SK_PROF_FF_ROWS = 15,  /* AFJLF pass 1 over the rows (reads the gradients) */
  SK_PROF_FF_RES = 16,   /* AFJLF residue pass and the layer sum             */
  SK_PROF_FF_SMALL = 17, /* AFJLF one-kernel layers (N' = D, forward)        */
  SK_PROF_FJL_T = 18,    /* FJL transpose in one pass (2^14 <= N' <= 2^21)   */
  SK_PROF_CLASSES = 19
};
#define SK_PROF_ALL ((1u << SK_PROF_CLASSES) - 1u)
int sketch_profile(sk_sketch *s, uint32_t classes);
int sketch_profile_read(sk_sketch *s, double *ms, int64_t *count, int64_t *bytes);

/* Thread-local message describing the last failure of this thread. */
const char *sketch_last_error(void);

/* Static text for a status code. */
const char *sketch_status_string(int code);

#ifdef __cplusplus
}
#endif

#endif /* SK_SKETCH_H */
