/*
 * lst.h -- C ABI of the exact large-sparse-target output-layer step on MI355X.
 *
 * The method (Vincent, de Brebisson, Bouthillier, "Efficient Exact Gradient
 * Update for training Deep Networks with Very Large Sparse Targets"):
 * a linear output layer o = W h with W of size D x d (D very large, d small),
 * trained against K-sparse targets y, is stepped WITHOUT forming the
 * D-dimensional output.  W is kept factored as W = V U (V: D x d, U: d x d,
 * section 3.2) together with Q = W^T W and U^{-T} (section 3.3), so that each
 * minibatch costs O(m d^2 + m^2 d + m^3) plus O(m K d) for the sparse rows of V
 * (minibatch algorithm, Appendix A), instead of O(m D d).
 *
 * Conventions shared by every entry point
 *   - All matrices are float32, row-major, densely packed (leading dimension =
 *     number of columns).  Indices are int32.
 *   - H is m x d: row i is the last hidden representation h_i of example i
 *     (the paper stores it as the i-th column of a d x m matrix; same bytes).
 *   - A target is given as K (index, value) pairs per example (section 2.1):
 *     Y_idx and Y_val are m x K; index -1 marks an unused slot (its value is
 *     ignored); an index that repeats inside one example adds its values.
 *   - Pointers documented "device" must be device memory of the GPU that was
 *     current when the state was created; "host" pointers are host memory.
 *   - Every call is asynchronous on the HIP stream given at creation, unless
 *     documented otherwise.  Caller-owned buffers must stay valid until that
 *     stream has executed the work.
 *   - Argument errors detected on the host are returned immediately and leave
 *     the state untouched.  Errors only the device can see (a target index
 *     outside [-1, D), a singular Woodbury matrix, a non-finite loss) are
 *     recorded in a sticky device flag: the step that raised it still writes
 *     loss and grad_H but skips every update of the state, and so does every
 *     later step until lst_sync() reports the error and clears the flag.
 *   - A state is not thread-safe; distinct states are independent.
 */
#ifndef LST_H
#define LST_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
enum {
  LST_OK = 0,
  LST_EINVAL = -1,      /* bad argument (null pointer, size, learning rate ...)   */
  LST_EINDEX = -2,      /* a target index outside [-1, D) (or -1 with the
                           spherical loss, which needs one class per example)    */
  LST_ESINGULAR = -3,   /* the m x m Woodbury matrix H^T H - A^{-1}/lr is
                           singular to working precision                          */
  LST_ENOMEM = -4,      /* device allocation failed                               */
  LST_EHIP = -5,        /* a HIP runtime call failed                              */
  LST_ENONFINITE = -6,  /* the loss of the minibatch is not finite                */
  LST_ESTATE = -7,      /* call not valid for this kind of state                  */
  LST_ENOSCRATCH = -8   /* larger than the static workspace of lst_stabilize_noalloc */
};

/* Loss functions (sections 3.1 and 3.6). */
enum {
  LST_LOSS_SQUARED = 0,   /* L_i = ||W h_i - y_i||^2                                    */
  LST_LOSS_SPHERICAL = 1, /* L_i = -log((o_c^2 + eps) / sum_j (o_j^2 + eps)), o = W h_i,
                             c = Y_idx[i][0] the target class; requires K == 1 and
                             ignores Y_val                                           */
  LST_LOSS_SPHERICAL_SHIFTED = 2
                          /* L_i = -log((o_c + eps)^2 / sum_j (o_j + eps)^2), the form
                             section 3.6 prints; K == 1, Y_val ignored.  Its gradient
                             moves every row of W along the all-ones direction, so a
                             factored state keeps W = V U + 1 c^T and s = W^T 1
                             (lst_get_shift); the minibatch steps then add O(m d) work
                             and one small launch between their second and third    */
};

typedef struct lst_config {
  int32_t loss;      /* LST_LOSS_SQUARED, LST_LOSS_SPHERICAL or LST_LOSS_SPHERICAL_SHIFTED */
  float sph_eps;     /* eps of the spherical softmax (> 0); unused for squared error   */
  int32_t m_max;     /* largest minibatch any lst_step call will pass (1..512)         */
  int32_t K_max;     /* largest K any lst_step call will pass (1..1024); m_max*K_max
                        must not exceed 16384 (lst_touched_rows orders the touched
                        rows of one step in one workgroup's LDS)                       */
  float cond_max;    /* drift control (Appendix C, pristine restore): after a step, if
                        ||U||_F * ||U^{-T}||_F > cond_max * d, set V <- V U, U <- I,
                        U^{-T} <- I (W and Q unchanged).  0 disables the check.      */
} lst_config;

typedef struct lst_state lst_state;

/* Statistics of a state (host copy; lst_stats synchronises the stream). */
typedef struct lst_stats_t {
  int64_t steps;           /* lst_step calls that were enqueued                        */
  int64_t restores;        /* pristine restores performed by drift control             */
  int32_t last_unique;     /* distinct target rows of the last factored step           */
  int32_t last_nnz;        /* valid (index, value) pairs of the last factored step     */
} lst_stats_t;

/*
 * lst_init -- create the factored state of section 3.2 / Appendix A.
 *   out   (host)   receives the new state; unchanged on error.
 *   D, d           output dimension (rows of W) and hidden size, D >= 1, 1 <= d <= 4096.
 *   V     (device) D x d initial V; copied, the caller keeps ownership.
 *   U     (device) d x d initial U, or NULL for the identity (the paper's
 *                  initialisation: V = W0, U = I).  Must be invertible.
 *   cfg   (host)   configuration, copied.
 *   hip_stream     hipStream_t every later call of this state is ordered on
 *                  (NULL = the default stream).
 * Computes U^{-T} (the identity when U is NULL) and Q = (V U)^T (V U); for
 * LST_LOSS_SPHERICAL_SHIFTED also s = (V U)^T 1, with c = 0.
 * Synchronous: returns after the state is ready.
 */
int lst_init(lst_state** out, int64_t D, int32_t d, const float* V, const float* U,
             const lst_config* cfg, void* hip_stream);

/*
 * lst_step -- one exact minibatch step (Appendix A, steps 1-10; for the
 * spherical softmax the same steps with the per-example loss derivatives).
 *   m, K            minibatch size (1..m_max) and pairs per example (1..K_max).
 *   H      (device) m x d hidden representations.
 *   Y_idx  (device) m x K target indices in [-1, D).
 *   Y_val  (device) m x K target values (ignored for the spherical loss).
 *   lr              learning rate eta > 0, finite.  The update is
 *                   W <- W - lr * dL/dW with L the SUM of the m per-example
 *                   losses (squared error: W <- W - 2 lr (W H - Y) H^T).
 *   loss   (device) m floats: per-example loss L_i.
 *   grad_H (device) m x d: row i = dL/dh_i (no 1/m factor).
 * Never forms W H.  State is updated in place unless the sticky error flag is set.
 * With m == 1 and K <= 256 the step takes the single-example form of
 * Algorithm 1 (Sherman-Morrison update of U^{-T}, eq. updateU-T) in two
 * launches; otherwise the minibatch steps of Appendix A.  Both compute the
 * same update in exact arithmetic, with the same error behaviour.
 */
int lst_step(lst_state* s, int32_t m, int32_t K, const float* H, const int32_t* Y_idx,
             const float* Y_val, float lr, float* loss, float* grad_H);

/*
 * lst_step_solve -- the same step as lst_step, with U^{-T} replaced by a solve
 * from scratch (section 3.5, last paragraph: for large m it can pay to solve
 * the d x d system with U_new each minibatch instead of keeping U^{-T} through
 * the m x m Woodbury inverse).  Per step: A = U_new^T is formed and factored
 * (partial pivoting), and U_new^T Z = H is solved for Z = U_new^{-T} H, which
 * gives the update of V (eq. updateV); Q and U move as in lst_step.  Same
 * arguments, outputs and device errors (LST_ESINGULAR: a zero pivot of U_new).
 * Requires d <= 1024 (LST_EINVAL otherwise).  Never captured into graphs; drift
 * control does not run (it needs U^{-T}).  Allocates its workspace (d^2 +
 * m_max d floats, 2 d ints) at the first call.  Afterwards the state's U^{-T}
 * no longer matches U: lst_step, lst_stabilize and lst_stabilize_noalloc
 * return LST_ESTATE until lst_restore (which sets U = U^{-T} = I).
 */
int lst_step_solve(lst_state* s, int32_t m, int32_t K, const float* H, const int32_t* Y_idx,
                   const float* Y_val, float lr, float* loss, float* grad_H);

/*
 * lst_materialize_W -- debug: W = V U (+ 1 c^T for LST_LOSS_SPHERICAL_SHIFTED)
 * into W (device, D x d).  O(D d^2).  For a naive state, copies its explicit W.
 */
int lst_materialize_W(lst_state* s, float* W);

/*
 * lst_get_shift -- debug: copy the shifted spherical loss's extra state of a
 * factored state (section 3.6): c (device, d floats; W = V U + 1 c^T) and
 * s = W^T 1 (device, d floats); either may be NULL.  States of the other
 * losses hold c = 0 and an s that is not kept up to date: LST_ESTATE.
 */
int lst_get_shift(lst_state* s, float* c, float* s_out);

/*
 * lst_get_state -- debug: copy Q, U and U^{-T} (each d x d, device; any may be
 * NULL) of a factored state.
 */
int lst_get_state(lst_state* s, float* Q, float* U, float* UinvT);

/* lst_get_V -- debug: copy V (device, D x d) of a factored state. */
int lst_get_V(lst_state* s, float* V);

/*
 * lst_touched_rows -- debug: the distinct target rows of the last factored
 * step in ascending order (the rows of V that step 9 of Appendix A updates).
 *   rows   (host) capacity m*K ints; receives the rows.
 *   count  (host) receives how many were written.
 * Synchronises the stream.
 */
int lst_touched_rows(lst_state* s, int32_t* rows, int32_t capacity, int32_t* count);

/*
 * lst_restore -- Appendix C pristine restore now: V <- V U, U <- I, U^{-T} <- I.
 * W = V U and Q are unchanged (up to rounding of V U).
 */
int lst_restore(lst_state* s);

/*
 * Appendix C, "stabilizing only problematic singular values": keep the
 * singular values of U inside a safe range [sigma_low, sigma_high] with
 * rank-one corrections that leave W = V U and Q unchanged, instead of the
 * O(D d^2) pristine restore.
 */
typedef struct lst_stab_config {
  float sigma_low;     /* safe range of the singular values of U; the appendix's   */
  float sigma_high;    /* example is [0.001, 100].  0 < sigma_low <= 1 <= sigma_high */
  int32_t squarings;   /* each estimate is 2^squarings power iterations (0..16; 7
                          gives 128, the appendix uses 100)                        */
  int32_t max_fixes;   /* at most this many corrections at each end of the spectrum
                          in one call (1..16)                                      */
  int32_t reinvert;    /* recompute U^{-T} from U: 0 never; 1 after each correction
                          (its rank-one update of U^{-T} cancels a term of size
                          1/sigma, costing about log10(1/sigma) digits in fp32);
                          2 also before the search, as the appendix does before
                          every check                                              */
} lst_stab_config;

typedef struct lst_stab_report {
  int32_t fixes_low;   /* singular values raised to 1 (they were below sigma_low)    */
  int32_t fixes_high;  /* singular values lowered to 1 (they were above sigma_high)  */
  float sigma_min;     /* estimate of sigma_min(U) made by the last round at the low
                          end (NaN if none ran); a value in range ended the rounds */
  float sigma_max;     /* the same at the high end                                  */
} lst_stab_report;

/*
 * lst_stabilize -- one run of the appendix's procedure on a factored state:
 *   1. if cfg->reinvert == 2, recompute U^{-T} from U (two Newton-Schulz steps
 *      Z <- 2Z - Z U^T Z from the current U^{-T}; they converge to the inverse
 *      whenever ||I - Z U^T|| < 1; in fp32 the result is accurate to about
 *      1e-7 cond(U), so with an ill-conditioned U prefer 1);
 *   2. estimate the smallest singular value of U and its left singular vector
 *      u by power iteration on U^{-T}; while it is below sigma_low (at most
 *      max_fixes times) apply fix-singular-value with target 1:
 *        alpha = (1 - sigma)/sigma, beta = -alpha/(1 + alpha),
 *        U <- U + alpha u (U^T u)^T,  V <- V + beta (V u) u^T,
 *        U^{-T} <- U^{-T} + beta u (U^{-1} u)^T;
 *   3. the same for the largest singular value (power iteration on U) against
 *      sigma_high.
 *   With cfg->reinvert >= 1, three Newton-Schulz steps follow every correction.
 * The power iteration starts from the vector of ones.  Every decision is taken
 * on the device; the call enqueues its kernels on the state's stream and, with
 * report == NULL, returns at once.  With report (host) it synchronises and
 * fills it.  Skipped (no change) when a step error is pending.  Allocates a
 * workspace of (2 + k) d^2 floats at its first call (k = split of the d^3 products).
 * Errors: LST_EINVAL for a null state or config or a config outside its ranges,
 * LST_ESTATE for a naive state, LST_ENOMEM, LST_EHIP.
 */
int lst_stabilize(lst_state* s, const lst_stab_config* cfg, lst_stab_report* report);

/*
 * lst_stabilize_noalloc -- lst_stabilize for callers that cannot allocate
 * device memory (code under HIP-graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the same kernels and results, but the workspace is a
 * static device array of 12 MiB that each GPU holds until the process ends,
 * instead of the state's workspace, which lst_stabilize allocates on first
 * use.  It fits d <= 512 with max_fixes <= 16; a larger problem returns
 * LST_ENOSCRATCH without doing anything.  Makes no allocation of any kind.
 * Every call on one GPU uses that GPU's array, which keeps the last call's
 * contents (each call initialises what it reads first): calls that overlap
 * on one GPU (two streams, two states) race and must be serialised by the
 * caller.  With report non-NULL the call synchronises the state's stream
 * (not capturable); pass NULL under capture.
 * Errors: as lst_stabilize, plus LST_ENOSCRATCH.
 */
int lst_stabilize_noalloc(lst_state* s, const lst_stab_config* cfg, lst_stab_report* report);

/*
 * lst_set_stabilize -- run lst_stabilize(cfg, NULL) after every `every`-th
 * lst_step (the appendix's n_check; 0 turns it off, the default).  With
 * HIP-graph replay the stabilisation runs outside the step's graph.
 */
int lst_set_stabilize(lst_state* s, int32_t every, const lst_stab_config* cfg);

/*
 * lst_naive_init -- explicit-W baseline state (sections 2.3 and 3.1: the
 * O(D d) per example computation the method avoids), same library, same GEMM
 * kernels.  W (device, D x d) is copied.  Synchronous.
 */
int lst_naive_init(lst_state** out, int64_t D, int32_t d, const float* W,
                   const lst_config* cfg, void* hip_stream);

/*
 * lst_naive_step -- same contract as lst_step, computed explicitly:
 * O = W H (D x m), residual / loss derivatives, grad_H = W^T dL/dO,
 * W <- W - lr dL/dO H^T.
 */
int lst_naive_step(lst_state* s, int32_t m, int32_t K, const float* H, const int32_t* Y_idx,
                   const float* Y_val, float lr, float* loss, float* grad_H);

/*
 * lst_set_graphs -- enable or disable (the default) HIP-graph replay of lst_step.
 * Replay lowers the host cost of a call; on MI355X it lengthens the step on
 * the device (the GPU idles between replays), so direct launches are the
 * default.  When enabled, the first lst_step call with a given argument tuple
 * (m, K, H, Y_idx, Y_val, lr, loss, grad_H) records its kernels into a graph and
 * every later call with the same tuple replays that graph with a single launch
 * on the state's stream (same kernels, same order, same results).  At most 32
 * graphs are kept; the least recently used is released first.  Profiling
 * (lst_profile_enable) bypasses the graphs.  Synchronises the stream and
 * releases the cached graphs.
 */
int lst_set_graphs(lst_state* s, int32_t enable);

/*
 * lst_set_split_tasks -- measurement aid for the minibatch step (Appendix A):
 * with enable != 0 every task that a launch of lst_step runs side by side (the
 * GEMM tiles, the target preparation and gather of V^T Y, Y^T Y, the per-example
 * scalars, the Woodbury solve, the scatter into V, the clear) runs as a launch
 * of its own, in the same order, so that a kernel trace or the profile phases
 * ("launch<L>.<task>") time each task alone.  The tasks of one launch are
 * independent: results are bitwise the same, the step is slower.  0 restores
 * the default.  Factored states only (LST_ESTATE otherwise); synchronises the
 * stream and releases the cached graphs.
 */
int lst_set_split_tasks(lst_state* s, int32_t enable);

/*
 * lst_sync -- wait for the state's stream; return and clear the sticky device
 * error (LST_OK if none).
 */
int lst_sync(lst_state* s);

/* lst_stats -- synchronise and fill *st. */
int lst_stats(lst_state* s, lst_stats_t* st);

/*
 * Profiling support for benchmarks.  While enabled, every lst_step brackets
 * each of its phases on the state's stream with a pair of HIP events (the
 * phases are listed by lst_profile_phase_name).  This adds event records to
 * the stream, so steps timed for throughput should run with profiling off.
 *   lst_profile_enable  enable != 0 turns it on, 0 off; either discards what
 *                       was recorded so far.
 *   lst_profile_read    synchronises, then writes the summed milliseconds of
 *                       each phase over the profiled steps into ms_total
 *                       (host, capacity doubles), the number of phases into
 *                       *nphases and of profiled steps into *nsteps; the
 *                       records are then discarded.
 */
int lst_profile_enable(lst_state* s, int32_t enable);
int lst_profile_read(lst_state* s, double* ms_total, int32_t capacity, int32_t* nphases,
                     int64_t* nsteps);
/* Name of phase i of lst_step (NULL when out of range). */
const char* lst_profile_phase_name(int32_t phase);

/*
 * The sparse input layer (section 2.2, "the easy part"): a D_in x d matrix
 * W_in whose input is K-sparse, given like the targets as K (index, value)
 * pairs per example (index -1 unused; a repeated index adds its values).
 * Only the rows the inputs refer to are read (forward) or written (update):
 * O(m K d) per minibatch instead of O(m D_in d).
 */
typedef struct lst_input lst_input;

/*
 * lst_input_init -- create an input layer; W_in (device, D_in x d) is copied.
 * D_in >= 1, 1 <= d <= 4096.  Besides W_in the layer holds a 1.8 MB table of
 * the rows of one update.  Synchronous.
 */
int lst_input_init(lst_input** out, int64_t D_in, int32_t d, const float* W_in,
                   void* hip_stream);

/*
 * lst_input_forward -- A = X W_in: row i of A (device, m x d) is
 * sum_k val[i][k] W_in[idx[i][k], :], the pairs added in k order (for K > 16:
 * in k order within each quarter of the list, the quarters then added in order).
 *   idx, val (device) m x K.  m, K >= 1, m * K <= 65536.
 * An index outside [-1, D_in) sets the sticky status LST_EINDEX (reported by
 * lst_input_sync) and its pair is left out of A.
 */
int lst_input_forward(lst_input* s, int32_t m, int32_t K, const int32_t* idx, const float* val,
                      float* A);

/*
 * lst_input_update -- W_in <- W_in - lr X^T grad_A (section 2.2: W_in[u_k] -=
 * lr v_k grad_a for every pair of every example; pairs that share a row add
 * up, in (example, pair) order, and each row is written once; a row named by
 * 64 or more pairs is summed in that order over each sixteenth of the m K
 * pairs, the sixteen sums then added in order).  grad_A
 * (device, m x d) is dL/dA.  lr > 0 and finite.  Rows no pair refers to are
 * not touched.  Skipped entirely (W_in unchanged) while the sticky status is
 * set, e.g. by an index outside [-1, D_in) in this call.
 */
int lst_input_update(lst_input* s, int32_t m, int32_t K, const int32_t* idx, const float* val,
                     const float* grad_A, float lr);

/* lst_input_get_W -- copy W_in into W (device, D_in x d). */
int lst_input_get_W(lst_input* s, float* W);

/* lst_input_sync -- wait for the stream; return and clear the sticky status. */
int lst_input_sync(lst_input* s);

/* lst_input_free -- synchronise and release the layer (NULL ok). */
void lst_input_free(lst_input* s);

/* lst_strerror -- static description of a status code. */
const char* lst_strerror(int status);

/* lst_free -- synchronise and release all device memory of the state (NULL ok). */
void lst_free(lst_state* s);

#ifdef __cplusplus
}
#endif

#endif /* LST_H */
