/*
 * sketch_hvp.h -- sketched Hessian-vector products and the Arnoldi iteration
 * in the sketched space (C ABI, same conventions as sketch.h).
 *
 * Sec. 2 of "Efficient Sketches for Training Data Attribution and Studying
 * the Loss Landscape" (Schioppa, NeurIPS 2024) sketches the HVP operator of a
 * loss as the map v -> S HVP(S^T v) of R^D to itself; the appendix "HVP in
 * implicit vs explicit form" describes the explicit evaluation used here: lift
 * v by S^T, apply the HVP in parameter space, sketch the result.  Sec. 4
 * ("Scaling eigenvalue estimation") runs Arnoldi with full
 * re-orthogonalisation on that map, so the stored Krylov basis has D entries
 * per vector instead of N.
 *
 * The HVP of a trained model needs the model and its data; this library
 * carries a synthetic Hessian with a known spectrum in their place:
 *
 *   H = shift I + sum_{j < r} lambda_j v_j v_j^T,   v_j = s_j / sqrt(N_tot),
 *
 * over the concatenated parameters of a layer list (N_tot = sum of the
 * layers' element counts; no padding).  s_j is a Rademacher vector
 * regenerated on the fly: coordinate e of layer l takes, for vector j, bit
 * (e mod 32) of word ((e / 32) mod 4) of the Philox4x32-10 block with counter
 * (lo32(e / 128), hi32(e / 128), (l << 6) | j, SK_STREAM_HVP) under the
 * key (lo32 seed, hi32 seed) of the Hessian's own seed; bit 1 means -1.  Its eigenvalues are
 * `shift` (multiplicity N_tot - r) and shift + eig(L^1/2 G L^1/2) with
 * L = diag(lambda), G = V^T V (a spike of r outliers over a flat bulk, the
 * structure the paper's Hessian-spectrum experiments look for).  Any other
 * HVP can be used with sketch_arnoldi_step, which only orthogonalises.  The
 * same Hessian defines the quadratic objective of the intrinsic-dimension
 * search below.
 *
 * Conventions: return 0 or a negative SK_E* code (sketch_last_error() gives
 * the message); device pointers are plain HIP addresses on the handle's
 * device; work is queued on `stream` (a hipStream_t, NULL = legacy default);
 * calls on one handle are serialised on one stream; no call after creation
 * allocates or frees device memory; results are bitwise deterministic.
 */
#ifndef SK_SKETCH_HVP_H
#define SK_SKETCH_HVP_H

#include <stdint.h>

#include "sketch.h"

#ifdef __cplusplus
extern "C" {
#endif

#define SK_STREAM_HVP 10 /* sign vectors s_j of the synthetic Hessian (fourth counter word) */
#define SK_HVP_MAX_RANK 32
#define SK_ARNOLDI_BREAKDOWN_TOL 1e-5f

typedef struct sk_hvp sk_hvp;

/*
 * Create the synthetic Hessian on `device`.
 *   shapes, n_layers  the parameter tensors (rows, cols >= 1; qk_* ignored);
 *                     the RNG layer index of shapes[i] is i.
 *   rank              r, 1 <= r <= SK_HVP_MAX_RANK.
 *   lambdas           host array of r fp32 spike weights.
 *   shift             the bulk eigenvalue.
 *   max_batch         most vectors one sk_hvp_apply / sketch_hvp call takes
 *                     (>= 1).  The handle owns sketch_hvp's workspace: two
 *                     buffers of max_batch N_tot floats (each layer's region
 *                     rounded up to 256 bytes).
 */
int sk_hvp_create(const sk_layer_shape *shapes, int32_t n_layers, int32_t rank, const float *lambdas, float shift,
                  uint64_t seed, int64_t max_batch, int32_t device, sk_hvp **out);

/*
 * y = H x for a batch of parameter vectors given per layer: x[i] and y[i]
 * (host arrays of n_layers device pointers) hold layer i as [batch, rows*cols]
 * fp32 row-major.  y may not alias x.  The pointers reach the kernels as a
 * small table copied to the device on `stream` (from pinned memory the
 * handle owns; a call waits for the previous call's copy before refilling
 * it).  Two passes, one launch each over all layers: the r inner products
 * s_j . x (fp32 per 8192-element chunk, chunks summed in fp64 in a fixed
 * order), then y = shift x + sum_j (lambda_j / N_tot)(s_j . x) s_j.
 * 1 <= batch <= max_batch.
 */
int sk_hvp_apply(sk_hvp *h, const float *const *x, int64_t batch, float *const *y, void *stream);

/* Free the handle (synchronises its device).  NULL is a no-op. */
void sk_hvp_destroy(sk_hvp *h);

/*
 * The sketched HVP operator (Sec. 2): out = S H S^T v for v [batch, D] fp32,
 * out [batch, D] fp32 (device).  `s` must have been created over the same
 * layer list as `h` (same count and element counts) and on the same device.
 * Runs sketch_apply_T into the handle's workspace, sk_hvp_apply, then
 * sketch_apply.  1 <= batch; batches above max_batch run in pieces.
 */
int sketch_hvp(sk_sketch *s, sk_hvp *h, const float *v, int64_t batch, float *out, void *stream);

/* Floats of caller workspace sketch_arnoldi_step needs for a basis of D-entry
 * vectors and Krylov dimension k (0 on bad arguments). */
int64_t sketch_arnoldi_work_floats(int64_t D, int32_t k);

/*
 * One step of Arnoldi with full re-orthogonalisation (Sec. 4), on a basis
 * Q [k+1, D] fp32 row-major (device) and Hbar [k+1, k] fp32 row-major
 * (device; column j is written whole by step j).
 *   j = -1   normalise row 0 of Q in place (a zero row stays zero).
 *   j >= 0   row j+1 holds w = A q_j on entry (the caller applied its
 *            operator, e.g. sketch_hvp); it is orthogonalised against rows
 *            0..j by two classical Gram-Schmidt passes (Hbar[0..j][j] = the
 *            sum of both passes' coefficients), then beta = |w| and
 *            Hbar[j+1][j] = beta, row j+1 = w / beta -- unless
 *            beta <= SK_ARNOLDI_BREAKDOWN_TOL |A q_j| (the Krylov space is
 *            exhausted to working precision), where both are set to 0.
 *            Hbar[j+2..k][j] = 0.  Requires j < k.
 *   work     device, sketch_arnoldi_work_floats(D, k) floats.
 */
int sketch_arnoldi_step(float *Q, int64_t D, int32_t j, float *Hbar, int32_t k, float *work, void *stream);

/*
 * k Arnoldi steps on the sketched synthetic HVP operator v -> S H S^T v from
 * v0 (device [D] fp32): Q [k+1, D] and Hbar [k+1, k] as above (device).  The
 * eigenvalues of Hbar[0:k, 0:k] (the Ritz values) estimate the extreme
 * eigenvalues of S H S^T.  The small k x k eigenproblem is the caller's: the
 * library stops at Hbar (the Python binding's ritz_values solves it with numpy
 * on the host).
 * The orthogonalisation scratch lives in the handle's workspace (it must hold
 * sketch_arnoldi_work_floats(D, k) floats, else SK_EUNSUPPORTED).
 */
int sketch_arnoldi(sk_sketch *s, sk_hvp *h, const float *v0, int32_t k, float *Q, float *Hbar, void *stream);

/*
 * Intrinsic-dimension search (Sec. 4, "Improving the search for the intrinsic
 * dimension", and the appendix listing of the search) on the synthetic
 * quadratic objective L(theta) = 1/2 theta^T H theta (minimum 0 at theta = 0)
 * with the metric tau = 1 - L(theta) / L(theta0), the fraction of the loss the
 * finetuning removes (the full model reaches 1).
 *   theta  = theta0 + S^T omega, omega in R^D (D = the sketch's D, the largest
 *            dimension allowed); only omega[0..d) is trained, the listing's
 *            zeroed gradient components.
 *   round  c steps of linear conjugate gradients on omega[0..d) (restarted
 *          from the current omega each round; gradient S H theta, Hessian
 *          S H S^T, one sketched HVP per step; a step with p.Mp <= 0 or r.r = 0
 *          changes nothing), then tau from the quadratic's expansion
 *          L = L0 + g0.omega + 1/2 omega.(S H S^T omega), g0 = S H theta0.
 *   rule   tau >= tau_target: done, res->d = d (status 0); else if the round
 *          improved tau by less than delta: d = 2 d, failing with status 1
 *          when d > D; status 2 when max_rounds rounds end undecided.
 *   theta0     host array of n_layers device pointers, fp32 [rows*cols].
 *   d_min      first d (1 <= d_min <= D); c, max_rounds >= 1.
 *   work       device, sketch_id_search_work_floats(D) floats; on return
 *              work[0..D) holds omega.
 *   tau_trace, d_trace  NULL or host arrays of max_rounds entries: tau and d
 *              of every round run.
 * Synchronises `stream` once per round to read tau (the decision is taken on
 * the host in double precision).
 */
typedef struct {
  int64_t d;       /* the estimate (0 unless status 0)                  */
  int32_t status;  /* 0 target reached, 1 D exceeded, 2 rounds exhausted */
  int32_t rounds;  /* rounds run                                          */
  double L0;       /* L(theta0)                                           */
} sk_id_result;
int64_t sketch_id_search_work_floats(int64_t D);
int sketch_id_search(sk_sketch *s, sk_hvp *h, const float *const *theta0, int64_t d_min, float tau_target,
                     float delta, int32_t c, int32_t max_rounds, float *work, double *tau_trace, int64_t *d_trace,
                     sk_id_result *res, void *stream);

/*
 * Kernel timing, as sketch_profile / sketch_profile_read, for the launches
 * this handle issues: class 0 = the inner-product pass of sk_hvp_apply (reads
 * x), class 1 = the combine pass (reads x, writes y), class 2 = Arnoldi
 * orthogonalisation kernels.  Arrays of SK_HVP_PROF_CLASSES entries.
 */
#define SK_HVP_PROF_CLASSES 3
int sk_hvp_profile(sk_hvp *h, uint32_t classes);
int sk_hvp_profile_read(sk_hvp *h, double *ms, int64_t *count, int64_t *bytes);

#ifdef __cplusplus
}
#endif

#endif /* SK_SKETCH_HVP_H */
