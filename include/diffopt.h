/*
 * diffopt.h -- C ABI of the MI355X (gfx950) differentiable-Adam hot path.
 *
 * The operations are those of TorchOpt (arXiv 2211.06934):
 *   - Sec. 2.3 "CPU/GPU-accelerated optimizers": the whole Adam optimizer is
 *     one differentiable operator with a hand-written forward and backward;
 *   - Listing 1 (explicit gradient): a non-inplace update + apply_updates,
 *     repeated for a number of inner steps, then one backward pass through
 *     all of them (the meta-gradient);
 *   - Sec. 2.3 "Memory-efficient and cache-friendly PyTree" and Appendix D,
 *     Table 2: tree flatten / unflatten of a parameter tree.
 * The paper prints no Adam formula; the update is Adam of Kingma & Ba (ICLR
 * 2015, Algorithm 1) with an extra eps_root inside the square root:
 *   t = count + 1,  c1 = 1 - b1^t,  c2 = 1 - b2^t
 *   m' = b1 m + (1-b1) g,   v' = b2 v + (1-b2) g^2
 *   s  = sqrt(v'/c2 + eps_root),   d = s + eps
 *   u  = -lr (m'/c1) / d,   p' = p + u
 *
 * Conventions shared by every call:
 *   - Element buffers are device pointers (HBM), fp32 unless stated, and
 *     owned by the caller; the library never allocates on these paths.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Calls enqueue work on it and return without synchronising; a fault in
 *     a kernel surfaces at the caller's next synchronisation.
 *   - Scalars cross the ABI in fp64; the library derives every coefficient
 *     (1-b1, 1-b2, 1/c1, 1/c2, lr/c1, ...) in fp64 and rounds each once to
 *     fp32 before the kernels use it.
 *   - Return value: DIFFOPT_OK or a negative code; the message for the last
 *     nonzero return on the calling thread is diffopt_last_error().  No call
 *     aborts the process or throws across the ABI.
 *   - n == 0 is a valid no-op.
 *   - 16-byte aligned element pointers take the 128-bit vector path; any
 *     other (4-byte aligned) pointer takes a scalar path with the same result.
 */
#ifndef DIFFOPT_H
#define DIFFOPT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DIFFOPT_OK 0
#define DIFFOPT_EINVAL (-1) /* bad argument: null pointer, range, overlap   */
#define DIFFOPT_ENOMEM (-2) /* host or device allocation failed             */
#define DIFFOPT_EHIP (-3)   /* a HIP runtime call or kernel launch failed   */

/* Longest run of unrolled steps whose moment trajectory the K-step backward
 * recomputes from one stored state (see diffopt_adam_unrolled_bwd).        */
#define DIFFOPT_REMAT_SPAN 8

/* Message describing the last nonzero return on this thread ("" if none);
 * error reporting of this ABI, not an operation of the paper.
 * The pointer stays valid until the next diffopt call on the same thread. */
const char* diffopt_last_error(void);

/* -------------------------------------------------------------------------
 * Segment table for tree flatten / unflatten (Appendix D, Table 2; Sec. 2.3
 * "PyTree").  A tree of S leaves maps onto one flat buffer: leaf j occupies
 * flat elements [off_j, off_j + numel_j), its elements in row-major order.
 *
 * The table depends only on the tree's structure (leaf sizes, layout and
 * element size), so one table serves every tree instance of that structure
 * (params, each step's grads, ...); leaf addresses are passed per call.
 */
typedef struct diffopt_segtable diffopt_segtable;

/* Build a table on the current HIP device (flatten/unflatten must run with
 * that device current; any other device gives EINVAL).
 *   nseg        number of leaves S (>= 0)
 *   numel       host array [nseg], elements per leaf (>= 0; empty leaves ok)
 *   offsets     host array [nseg] of flat element offsets, or NULL for the
 *               dense layout off_j = numel_0 + ... + numel_{j-1}.  Explicit
 *               offsets may leave gaps (untouched by flatten) but the flat
 *               ranges of nonempty leaves must not overlap (EINVAL).
 *   elem_bytes  element size in bytes: 1, 2, 4 or 8 (fp32 = 4)
 *   out         receives the table; the caller frees it with
 *               diffopt_segtable_destroy.
 * Copies what it needs; the caller's arrays may be freed on return.  Owns a
 * small device array (about 32 bytes per nonempty leaf), uploaded
 * synchronously here.                                                      */
int diffopt_segtable_create(int64_t nseg, const int64_t* numel,
                            const int64_t* offsets, int32_t elem_bytes,
                            diffopt_segtable** out);

/* Free a table and its device memory (NULL is a no-op).  The caller must
 * make sure no enqueued call still uses it, and must not destroy a table
 * while a stream is being captured into a graph (freeing device memory is
 * not a capturable operation).  (The table is the tree structure of
 * Sec. 2.3 "PyTree", kept on the device.)                                   */
void diffopt_segtable_destroy(diffopt_segtable* table);

/* Flat length n in elements of the flattened tree (Sec. 2.3 "PyTree"): the
 * max over leaves of off_j + numel_j; -1 if
 * table is NULL.                                                            */
int64_t diffopt_segtable_total(const diffopt_segtable* table);

/* Number of leaves S the table was built for (Sec. 2.3 "PyTree"); -1 if
 * table is NULL.                                                            */
int64_t diffopt_segtable_nseg(const diffopt_segtable* table);

/* Tree flatten (pack; Appendix D, Table 2 "Tree Flatten"):
 * flat[off_j + i] = leaf_j[i] for all j, i < numel_j.
 *   leaf_ptrs   DEVICE array [nseg] of uint64 leaf addresses, in table order
 *               (entries of empty leaves are ignored and may be 0)
 *   flat        device buffer of at least diffopt_segtable_total() elements
 * Copies bits through integer registers: NaN payloads, signed zeros and
 * subnormals survive.  Pointers must be aligned to elem_bytes.  The flat
 * buffer must not overlap any leaf.  Small tables (at most 32 nonempty
 * leaves and 65,536 elements, laid out as the plain concatenation of the
 * leaves) are copied one element per lane with the table in the kernel
 * arguments; the result is the same.                                       */
int diffopt_tree_flatten(const diffopt_segtable* table,
                         const uint64_t* leaf_ptrs, void* flat, void* stream);

/* Tree unflatten (unpack; Appendix D, Table 2 "Tree UnFlatten"), the mirror:
 * leaf_j[i] = flat[off_j + i].
 * Leaves must not overlap each other or the flat buffer.                     */
int diffopt_tree_unflatten(const diffopt_segtable* table, const void* flat,
                           const uint64_t* leaf_ptrs, void* stream);

/* Batched forms: ntrees trees of the same structure (one table) in one
 * launch per 16 trees, e.g. the params tree and the K gradient trees of an
 * unrolled inner loop (Listing 1 flattens each of them).  Tree t is
 * leaf_ptrs[t] (a DEVICE array [nseg] of leaf addresses, as above) and
 * flats[t] (its flat buffer); leaf_ptrs and flats are HOST arrays [ntrees].
 * The result equals ntrees calls of diffopt_tree_flatten /
 * diffopt_tree_unflatten; no tree may overlap another tree's buffers.
 * ntrees == 0 is a no-op.                                                   */
int diffopt_tree_flatten_batch(const diffopt_segtable* table, int64_t ntrees,
                               const uint64_t* const* leaf_ptrs,
                               void* const* flats, void* stream);

int diffopt_tree_unflatten_batch(const diffopt_segtable* table, int64_t ntrees,
                                 const void* const* flats,
                                 const uint64_t* const* leaf_ptrs, void* stream);

/* -------------------------------------------------------------------------
 * Differentiable Adam step, forward (Sec. 2.3; Listing 1's
 * opt.update(..., inplace=False) followed by apply_updates, fused).
 *   params, grad, mu, nu        inputs [n]
 *   count                       steps already taken (>= 0); bias correction
 *                               uses t = count + 1; the caller's state
 *                               becomes count + 1
 *   lr (finite), b1, b2 in [0, 1), eps >= 0, eps_root >= 0
 *   params_out, mu_out, nu_out  outputs [n] (p', m', v')
 *   update_out                  optional output [n] (u = p' - p), or NULL
 * Each output may alias its own input (params_out == params, ...): every
 * element is read and then written by one thread.  Writing mu_out/nu_out
 * over mu/nu destroys what diffopt_adam_bwd needs: that is the
 * non-differentiable in-place mode.                                         */
int diffopt_adam_fwd(const float* params, const float* grad, const float* mu,
                     const float* nu, int64_t n, int64_t count, double lr,
                     double b1, double b2, double eps, double eps_root,
                     float* params_out, float* mu_out, float* nu_out,
                     float* update_out, void* stream);

/* Differentiable Adam step, backward: the vector-Jacobian product of
 * diffopt_adam_fwd (Sec. 2.3: hand-written backward with symbolic reduction
 * and explicit cancelling of 0/0 cases).
 *   dupdate    cotangent of params_out [n] (equal to that of update_out,
 *              since params_out = params + update)
 *   dmu, dnu   cotangents of mu_out, nu_out [n], or NULL for zero
 *   grad, mu, nu   the forward's INPUTS g, m, v (not its outputs)
 *   count, lr, b1, b2, eps, eps_root   as passed to the forward
 *   dparams    cotangent of params [n]; the params path is the identity, so
 *              this is a copy of dupdate; NULL (or == dupdate) skips it
 *   dgrad, dmu_in, dnu_in   cotangents of grad, mu, nu [n]
 * dmu_in may alias dmu and dnu_in may alias dnu (read-then-write per
 * element).  The computation is the algebraically reduced form, in which
 * the g^2 terms of the plain chain rule cancel exactly:
 *   a = (1-b1)/c1,  b = (1-b2)/c2
 *   N = b b1 g m / c1 - a b2 v / c2 - a (eps_root + s eps)
 *   dgrad  = (1-b1) dmu + 2 (1-b2) g dnu + dupdate lr N / (s d^2)
 *   dmu_in = b1 (dmu - dupdate lr / (c1 d))
 *   dnu_in = b2 (dnu + dupdate lr (m'/c1) / (2 c2 s d^2))
 * At s == 0 (only when eps_root == 0, v == 0 and g == 0) the dupdate term of
 * dgrad is -dupdate lr a / d (the two-sided mean derivative) and that of
 * dnu_in is 0.                                                              */
int diffopt_adam_bwd(const float* dupdate, const float* dmu, const float* dnu,
                     const float* grad, const float* mu, const float* nu,
                     int64_t n, int64_t count, double lr, double b1, double b2,
                     double eps, double eps_root, float* dparams, float* dgrad,
                     float* dmu_in, float* dnu_in, void* stream);

/* -------------------------------------------------------------------------
 * K-step unrolled driver, forward (Listing 1's inner loop with the K
 * gradients given up front):
 *   for k = 1..K: (p_k, mu_k, nu_k) = adam_fwd(p_{k-1}, grads[k-1],
 *                                             mu_{k-1}, nu_{k-1}, count0+k-1)
 *   K >= 1, n >= 0
 *   p0          input [n] (not modified unless pK == p0)
 *   grads       HOST array [K] of device pointers, grads[k-1] = g_k
 *   mu_traj     HOST array [K+1] of device pointers: mu_traj[0] = mu0 is
 *               read, mu_traj[k] receives mu_k.  mu_traj[0] and mu_traj[K]
 *               (the final state) are required; an intermediate entry
 *               (0 < k < K) may be NULL, and that state is then not stored
 *               (the backward recomputes it, see below).  Non-NULL entries
 *               are distinct buffers
 *   nu_traj     the same for nu; nu_traj[k] is NULL exactly when mu_traj[k]
 *               is
 *   pK          output [n] (may equal p0)
 * grads, the stored mu_traj[1..K], nu_traj[1..K] and pK must not overlap one
 * another or p0, mu_traj[0], nu_traj[0] (pK == p0 excepted).
 * The K steps run fused, one kernel per 16 steps: each element's running
 * params and moments stay in registers between steps, so K steps move
 * 16 + 4K + 8 S bytes per element for S stored states (16 + 12K with the
 * whole trajectory, 24 + 4K with the final state only).  When a 16-step
 * launch boundary falls on an unstored state, the running moments pass to the
 * next launch through mu_traj[K], nu_traj[K].  Every stored state and pK
 * equal K calls of diffopt_adam_fwd bit for bit.  Pointers that are not
 * 16-byte aligned take a one-element-per-lane kernel with the same result.
 * No host synchronisation.                                                  */
int diffopt_adam_unrolled_fwd(int64_t K, int64_t n, const float* p0,
                              const float* const* grads,
                              float* const* mu_traj, float* const* nu_traj,
                              float* pK, int64_t count0, double lr, double b1,
                              double b2, double eps, double eps_root,
                              void* stream);

/* K-step unrolled driver, backward (the meta-gradient of Listing 1's final
 * autograd.grad): starting from the cotangent dpK of p_K and zero
 * cotangents of mu_K, nu_K,
 *   for k = K..1: (dP, dgrads[k-1], dM, dV) = adam_bwd(dP, dM, dV, g_k,
 *                                   mu_{k-1}, nu_{k-1}, count0+k-1)
 *   dpK         input [n]; the cotangent of p0 equals dpK (identity), so it
 *               is not copied
 *   grads, mu_traj, nu_traj   as given to / written by the forward (HOST
 *               arrays of device pointers; mu_traj[K], nu_traj[K] unused).
 *               A NULL intermediate entry k is recomputed from the latest
 *               stored state j < k and g_{j+1..k} with the forward's own
 *               recurrences, so the result is the same bit for bit; at most
 *               DIFFOPT_REMAT_SPAN - 1 consecutive entries may be NULL
 *               (EINVAL otherwise, before anything is enqueued)
 *   dgrads      HOST array [K] of device pointers: dgrads[k-1] receives the
 *               cotangent of g_k
 *   dmu0, dnu0  outputs [n]: cotangents of mu0, nu0 (also the running dM,
 *               dV between launches)
 * Outputs must not overlap the inputs or one another.
 * The K steps run fused, last step first, with each element's dM, dV in
 * registers: a run of steps whose input states are stored takes one launch
 * per 16 steps and reads each state back (12 + 16K bytes per element for
 * the whole trajectory); a run of C <= DIFFOPT_REMAT_SPAN steps after one
 * stored state takes one launch that reads that state and the C gradients
 * once, recomputes the run's states in registers, then runs its VJP steps
 * (20 + 8K bytes per element for K <= DIFFOPT_REMAT_SPAN with nothing
 * stored).  The result equals K calls of diffopt_adam_bwd (the first with
 * zero dM, dV) on the full trajectory bit for bit.  Pointers that are not
 * 16-byte aligned take one-element-per-lane kernels with the same result. */
int diffopt_adam_unrolled_bwd(int64_t K, int64_t n, const float* dpK,
                              const float* const* grads,
                              const float* const* mu_traj,
                              const float* const* nu_traj,
                              float* const* dgrads, float* dmu0, float* dnu0,
                              int64_t count0, double lr, double b1, double b2,
                              double eps, double eps_root, void* stream);


/* -------------------------------------------------------------------------
 * Leaf-direct ("tree map") form of the differentiable Adam step (Appendix D,
 * Table 2 "Tree Map"; Sec. 2.3 for the step): the same forward and VJP as
 * diffopt_adam_fwd / diffopt_adam_bwd applied to every leaf of parameter
 * trees, reading and writing the leaves themselves, so no flatten or
 * unflatten is needed.  The result equals flatten -> flat step -> unflatten
 * element for element.
 *   table       a segment table with elem_bytes == 4 describing the leaf
 *               sizes (its flat offsets are not used); the current device
 *               must be the table's
 *   every other pointer argument is a DEVICE array [nseg] of uint64 leaf
 *               addresses of one operand tree, in table order (entries of
 *               empty leaves are ignored); leaves are fp32, 4-byte aligned;
 *               leaves 16-byte aligned in every operand take 128-bit
 *               accesses, others an element path with the same result
 * Aliasing as in the flat calls: an output leaf may be its own input leaf
 * (params_out[j] == params[j], dmu_in[j] == dmu[j], ...), never another leaf.
 * dmu and dnu are both NULL (zero cotangents) or both given.
 * Small trees (at most 32 nonempty leaves and 65,536 elements) run one
 * element per lane with the leaf table in the kernel arguments; the results
 * are the same bit for bit.                                                */
int diffopt_adam_fwd_tree(const diffopt_segtable* table, const uint64_t* params,
                          const uint64_t* grad, const uint64_t* mu,
                          const uint64_t* nu, int64_t count, double lr,
                          double b1, double b2, double eps, double eps_root,
                          const uint64_t* params_out, const uint64_t* mu_out,
                          const uint64_t* nu_out, void* stream);

int diffopt_adam_bwd_tree(const diffopt_segtable* table, const uint64_t* dupdate,
                          const uint64_t* dmu, const uint64_t* dnu,
                          const uint64_t* grad, const uint64_t* mu,
                          const uint64_t* nu, int64_t count, double lr,
                          double b1, double b2, double eps, double eps_root,
                          const uint64_t* dgrad, const uint64_t* dmu_in,
                          const uint64_t* dnu_in, void* stream);

/* K-step unrolled driver in leaf-direct form (Listing 1's loop; Appendix D,
 * Table 2 "Tree Map"): the recurrences of
 * diffopt_adam_unrolled_fwd / _bwd with every flat buffer replaced by a tree
 * (a device array of leaf addresses).  grads, mu_traj, nu_traj and dgrads are
 * HOST arrays ([K], [K+1], [K+1], [K]) of such device arrays.  The steps run
 * fused, one kernel per 8 steps, each lane keeping its elements' running
 * params (forward) or dM, dV (backward) in registers: 16 + 12K and 12 + 16K
 * bytes per element, and results equal to K calls of the single-step
 * leaf-direct entry points bit for bit.  pK may be p0; dmu0 / dnu0 also carry
 * the running cotangents between launches when K > 8.  Output leaves must
 * not overlap input leaves or one another.                                  */
int diffopt_adam_unrolled_fwd_tree(const diffopt_segtable* table, int64_t K,
                                   const uint64_t* p0,
                                   const uint64_t* const* grads,
                                   const uint64_t* const* mu_traj,
                                   const uint64_t* const* nu_traj,
                                   const uint64_t* pK, int64_t count0, double lr,
                                   double b1, double b2, double eps,
                                   double eps_root, void* stream);

int diffopt_adam_unrolled_bwd_tree(const diffopt_segtable* table, int64_t K,
                                   const uint64_t* dpK,
                                   const uint64_t* const* grads,
                                   const uint64_t* const* mu_traj,
                                   const uint64_t* const* nu_traj,
                                   const uint64_t* const* dgrads,
                                   const uint64_t* dmu0, const uint64_t* dnu0,
                                   int64_t count0, double lr, double b1,
                                   double b2, double eps, double eps_root,
                                   void* stream);

/* -------------------------------------------------------------------------
 * The paper's other fused differentiable optimizers (Sec. 1, contribution
 * (2)(i): SGD, RMSProp, Adam; Sec. 2.3).  The paper prints no formula; these
 * are the textbook forms as torch.optim implements them.  Conventions as for
 * Adam: fp32 device buffers [n], scalars in fp64, n == 0 is a no-op, outputs
 * may alias their own inputs, state buffers that are NULL read as zero.
 *
 * SGD with momentum mu >= 0 (trace t):
 *   t' = mu t + g;  u = -lr t'  (nesterov != 0: u = -lr (g + mu t'));  p' = p + u
 *   mu == 0 is plain SGD: trace and trace_out are ignored (may be NULL).
 *   mu  > 0: trace may be NULL (zero, the first step); trace_out required.  */
int diffopt_sgd_fwd(const float* params, const float* grad, const float* trace,
                    int64_t n, double lr, double momentum, int32_t nesterov,
                    float* params_out, float* trace_out, void* stream);

/* VJP of diffopt_sgd_fwd (Sec. 2.3: hand-written backward).  dparams_out:
 * cotangent of p' (the cotangent of p
 * is the same array); dtrace_out: cotangent of t' (NULL = zero).  Writes the
 * cotangent of g and, when mu > 0, of t (dtrace_in, required then).  The map
 * is linear, so no forward input is needed.                               */
int diffopt_sgd_bwd(const float* dparams_out, const float* dtrace_out,
                    int64_t n, double lr, double momentum, int32_t nesterov,
                    float* dgrad, float* dtrace_in, void* stream);

/* RMSProp (Sec. 1, contribution (2)(i)) with decay alpha in [0, 1), eps >= 0
 * outside and eps_root >= 0
 * inside the root, momentum mu >= 0 (buffer b):
 *   v' = alpha v + (1-alpha) g^2;  d = sqrt(v' + eps_root) + eps
 *   mu == 0: u = -lr g / d          (mom, mom_out ignored)
 *   mu  > 0: b' = mu b + g / d, u = -lr b'   (mom may be NULL; mom_out required)
 *   p' = p + u                                                             */
int diffopt_rmsprop_fwd(const float* params, const float* grad, const float* nu,
                        const float* mom, int64_t n, double lr, double alpha,
                        double eps, double eps_root, double momentum,
                        float* params_out, float* nu_out, float* mom_out,
                        void* stream);

/* VJP of diffopt_rmsprop_fwd (Sec. 2.3: hand-written backward, symbolic
 * reduction, explicit 0/0 cases), in the algebraically reduced form (the g^2
 * terms of the chain rule cancel).  Cotangents of p', v', b' (dnu_out and
 * dmom_out may be NULL = zero); grad and nu are the forward's INPUTS.
 * Writes the cotangents of g, v and, when mu > 0, of b (dmom_in required).
 * At the 0/0 point (eps_root = 0, v = 0, g = 0) the update's contribution to
 * dg is the two-sided mean derivative and its contribution to dv is 0.    */
int diffopt_rmsprop_bwd(const float* dparams_out, const float* dnu_out,
                        const float* dmom_out, const float* grad,
                        const float* nu, int64_t n, double lr, double alpha,
                        double eps, double eps_root, double momentum,
                        float* dgrad, float* dnu_in, float* dmom_in,
                        void* stream);

/* Leaf-direct ("tree map") forms of the four calls above (Appendix D,
 * Table 2 "Tree Map"): the same arithmetic applied to every leaf of
 * parameter trees, one launch each, with the conventions of the leaf-direct
 * Adam calls (a table with elem_bytes == 4 on the current device; every other
 * pointer a DEVICE array [nseg] of fp32 leaf addresses in table order, NULL
 * where the flat call takes NULL; an output leaf may be its own input leaf).
 * The result equals flatten -> flat call -> unflatten element for element. */
int diffopt_sgd_fwd_tree(const diffopt_segtable* table, const uint64_t* params,
                         const uint64_t* grad, const uint64_t* trace,
                         double lr, double momentum, int32_t nesterov,
                         const uint64_t* params_out, const uint64_t* trace_out,
                         void* stream);

int diffopt_sgd_bwd_tree(const diffopt_segtable* table,
                         const uint64_t* dparams_out, const uint64_t* dtrace_out,
                         double lr, double momentum, int32_t nesterov,
                         const uint64_t* dgrad, const uint64_t* dtrace_in,
                         void* stream);

int diffopt_rmsprop_fwd_tree(const diffopt_segtable* table,
                             const uint64_t* params, const uint64_t* grad,
                             const uint64_t* nu, const uint64_t* mom,
                             double lr, double alpha, double eps,
                             double eps_root, double momentum,
                             const uint64_t* params_out, const uint64_t* nu_out,
                             const uint64_t* mom_out, void* stream);

int diffopt_rmsprop_bwd_tree(const diffopt_segtable* table,
                             const uint64_t* dparams_out,
                             const uint64_t* dnu_out, const uint64_t* dmom_out,
                             const uint64_t* grad, const uint64_t* nu,
                             double lr, double alpha, double eps,
                             double eps_root, double momentum,
                             const uint64_t* dgrad, const uint64_t* dnu_in,
                             const uint64_t* dmom_in, void* stream);

/* -------------------------------------------------------------------------
 * Zero-order (evolution-strategies) gradient estimation (Sec. 2.2
 * "Zero-order Differentiation"): grad f_s(theta) = (1/s) E_z[f(theta + s z) z]
 * for the Gaussian smoothing f_s(theta) = E_z[f(theta + s z)], z ~ N(0, I),
 * estimated by Monte-Carlo over N noise vectors that the caller draws.
 *
 * es_perturb: the points at which the caller evaluates f.
 *   params      theta [n]
 *   noise       [num_samples][n], row-major (row i is z_i)
 *   out         [num_samples][n], row i = theta + sigma z_i; with antithetic != 0
 *               [2 num_samples][n], rows num_samples + i = theta - sigma z_i
 * num_samples <= 65,535 x 8.  n % 4 == 0 with 16-byte aligned pointers takes
 * 128-bit accesses; anything else an element path with the same result.    */
int diffopt_es_perturb(const float* params, const float* noise,
                       int64_t num_samples, int64_t n, double sigma,
                       int32_t antithetic, float* out, void* stream);

/* es_estimate (Sec. 2.2, the Monte-Carlo estimate of the smoothed gradient):
 * grad_j = scale * sum_i weights_i noise_ij, accumulated in
 * sample order in fp32.  weights is a DEVICE array [num_samples] formed by the
 * caller from its evaluations f_i:
 *   plain:       w_i = f(theta + s z_i),                    scale = 1/(N s)
 *   baseline:    w_i = f(theta + s z_i) - f(theta),         scale = 1/(N s)
 *   antithetic:  w_i = f(theta + s z_i) - f(theta - s z_i), scale = 1/(2 N s)
 * num_samples == 0 writes zeros.                                            */
int diffopt_es_estimate(const float* noise, const float* weights,
                        int64_t num_samples, int64_t n, double scale,
                        float* grad, void* stream);

/* The same two steps with the Gaussian noise generated inside the kernels
 * (Sec. 2.2; Listing 3 makes the noise sampler part of the estimator): no
 * noise array exists.  z_ij, for sample i < num_samples and parameter
 * j < n, is a pure function of (seed, i, j):
 *   slot   = with q = j mod 512: block c = 64 (j / 512) + (q mod 256) / 4,
 *            word w = 2 (q / 256) + (q mod 4) / 2, and the cosine normal for
 *            even q, the sine one for odd q (so block c covers two runs of
 *            four parameters 256 apart, and 64 consecutive blocks fill two
 *            contiguous 1 KiB runs);
 *   block  = Philox-4x64-10 (Salmon, Moraes, Dror, Shaw, SC 2011) of the
 *            counter (c, i, 0, 0) under the key (seed, 0): four 64-bit
 *            words;
 *   word   = word w of the block, split into its low and high 32 bits lo, hi;
 *   u1     = (floor(lo / 2^8) + 1) 2^-24 in (0, 1], u2 = floor(hi / 2^8) 2^-24
 *            in [0, 1);
 *   z_ij   = sqrt(-2 ln u1) cos(2 pi u2) for even q, sqrt(-2 ln u1)
 *            sin(2 pi u2) for odd q (Box and Muller, 1958), computed in fp32
 *            with the hardware log2, square root, sine and cosine: within
 *            3.5e-7 r of the exact value, r = sqrt(-2 ln u1) (measured over
 *            every value the two uniforms can take).
 * The same seed gives the same z in both calls, and in any launch shape.
 *
 * es_perturb_gaussian: out as for diffopt_es_perturb ([N][n], or [2N][n]
 *   with antithetic != 0); num_samples <= 65,535 x 8.  n % 4 == 0 with
 *   16-byte aligned pointers takes 128-bit accesses, anything else an element
 *   path with the same result.
 * es_estimate_gaussian: grad_j = scale * sum_i w_i z_ij, accumulated in
 *   sample order in fp32, with the weights and scale formed in the kernel
 *   from the caller's evaluations `fvals` (a DEVICE array):
 *     method 0, plain:      w_i = f_i,            scale = 1/(N s), fvals [N]
 *     method 1, baseline:   w_i = f_i - *f0,      scale = 1/(N s), fvals [N],
 *                           f0 a DEVICE pointer to f(theta)
 *     method 2, antithetic: w_i = f_i - f_{N+i},  scale = 1/(2 N s), fvals [2N]
 *                           (the evaluations of the rows es_perturb_gaussian
 *                           wrote, in order)
 *   scale is formed in fp64 and rounded once.  sigma must be finite and
 *   nonzero; num_samples == 0 writes zeros.                              */
int diffopt_es_perturb_gaussian(const float* params, int64_t n,
                                int64_t num_samples, uint64_t seed,
                                double sigma, int32_t antithetic, float* out,
                                void* stream);
int diffopt_es_estimate_gaussian(const float* fvals, const float* f0,
                                 int64_t num_samples, int32_t method,
                                 int64_t n, uint64_t seed, double sigma,
                                 float* grad, void* stream);

/* es_weights: weights[i] = scale * w_i, the method's weights and scale as in
 * diffopt_es_estimate_gaussian, for diffopt_es_estimate with scale 1 (a
 * caller that draws its own noise, e.g. from another distribution).  DEVICE
 * arrays; num_samples == 0 is a no-op.                                    */
int diffopt_es_weights(const float* fvals, const float* f0,
                       int64_t num_samples, int32_t method, double sigma,
                       float* weights, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DIFFOPT_H */
