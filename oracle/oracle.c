/*
 * oracle.c -- plain CPU reference for the differentiable Adam step, its
 * vector-Jacobian product, the K-step unrolled driver and tree pack/unpack.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the oracle the GPU path is tested
 * against.  Only the test-suite, the smoke check and the CPU-baseline leg of
 * the benchmark may load it.  It shares no source, header, table or helper
 * with the HIP library, and the HIP library never calls it.
 *
 * Conventions:
 *   - fp64 everywhere; callers upcast fp32 inputs element by element (exact).
 *   - single thread, scalar loops, no blocking, no fusion beyond the
 *     definition; built with -O2 -ffp-contract=off and without -ffast-math,
 *     so every operation is a separately rounded IEEE double operation.
 *
 * What the paper fixes and what it does not (TorchOpt, arXiv 2211.06934):
 *   - Sec. 2.3 "CPU/GPU-accelerated optimizers": Adam is treated as ONE
 *     differentiable operator with a hand-written forward and backward, and
 *     some 0/0 cases are cancelled explicitly.  The paper prints no Adam
 *     formula.  The forward below is Adam as defined by Kingma & Ba (ICLR
 *     2015, Algorithm 1), with an extra eps_root term inside the square root
 *     (eps_root = 0 gives the textbook update).
 *   - Listing 1 (explicit gradient, functional API): a non-inplace update
 *     followed by apply_updates, repeated for iter_times steps, then one
 *     backward pass through all of them.  The unrolled driver below is that
 *     loop with the gradients supplied from outside.
 *   - Sec. 2.3 "Memory-efficient and cache-friendly PyTree" and Appendix D,
 *     Table 2 ("Tree Flatten", "Tree UnFlatten"): flattening a tree into one
 *     buffer and splitting it back.  pack/unpack below are the definition:
 *     leaf j occupies flat elements [off_j, off_j + numel_j), row-major.
 *
 * Readings where the paper is silent (each also listed in the design notes):
 *   R1  count = number of steps already taken; bias correction uses
 *       t = count + 1, c1 = 1 - b1^t, c2 = 1 - b2^t.
 *   R2  params_out = params + update (apply_updates fused into the step);
 *       the cotangent of the update equals the cotangent of params_out.
 *   R3  the 0/0 case: s = sqrt(v_hat + eps_root) = 0 happens only when
 *       eps_root = 0, v = 0 and g = 0.  There the P-bar contribution to the
 *       nu cotangent is defined as 0.  The resulting d/dg is the symmetric
 *       (two-sided mean) derivative of the update at g = 0.
 *
 * Parity pins (tests that tie this file to something other than itself):
 *   forward : step-1 closed form; constant-gradient bias-correction invariant;
 *             b1 = b2 = 0 special case; gradient-scale invariance;
 *             torch.optim.Adam in fp64 at eps_root = 0 over many steps.
 *   backward: step-1 closed form; linearity in the cotangents; autograd
 *             through torch.optim's functional Adam (differentiable mode) in
 *             fp64; fp64 central differences of the forward, including the
 *             symmetric difference at g = 0 (reading R3) and, from a fresh
 *             state (m = 0), the one-sided difference in v there, which is
 *             exactly 0 since the update vanishes for every v >= 0.
 *   unrolled: fp64 central differences of the K-step map.
 *   pack    : numpy concatenation, bit for bit; unpack(pack(x)) == x.
 *   noise   : Philox-4x64-10 bit for bit against numpy's independent
 *             implementation (numpy.random.Philox); the Box-Muller transform
 *             against its closed-form values (u1 = 1, u1 = 2^-k at the angles
 *             0, pi/4, pi/2, pi, 3 pi/2); the composed noise against the
 *             standard normal (moments, Kolmogorov-Smirnov, tails) and the
 *             independence of each element from N and n.
 *   ES      : exact recovery of linear and quadratic gradients with a
 *             symmetric orthonormal sample set, for every weighting method.
 *   mag_*   : the tolerance scales are sums of absolute values of terms.
 *             From below they bound |value| (triangle inequality); from
 *             above they equal |value| on inputs whose terms all share one
 *             sign, and copies of this file with any one term doubled are
 *             built and shown to fail that equality.
 *
 * Accuracy limit of the plain chain rule: the update's two dg terms (and
 * RMSProp's) are each of size lr a / s and cancel exactly when the state is
 * fresh and eps = eps_root = 0, so with a tiny s their fp64 difference keeps
 * a rounding residue of about 1e-16 lr a / s instead of 0.  Tests in that
 * regime take dg from the closed form (the update is constant in g there).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>

/* Bias-correction denominators, reading R1. */
static void bias_corrections(int64_t count, double b1, double b2,
                             double* c1, double* c2) {
  double t = (double)(count + 1);
  *c1 = 1.0 - pow(b1, t);
  *c2 = 1.0 - pow(b2, t);
}

/*
 * One Adam step (Kingma & Ba, Algorithm 1; reading R2 for params_out),
 * element by element:
 *   m' = b1 m + (1-b1) g            v' = b2 v + (1-b2) g^2
 *   m^ = m'/c1                      v^ = v'/c2
 *   s  = sqrt(v^ + eps_root)        d  = s + eps
 *   u  = -lr m^ / d                 p' = p + u
 * u_out may be NULL.
 */
void oracle_adam_fwd(int64_t n, const double* p, const double* g,
                     const double* m, const double* v, int64_t count,
                     double lr, double b1, double b2, double eps,
                     double eps_root, double* p_out, double* m_out,
                     double* v_out, double* u_out) {
  double c1, c2;
  bias_corrections(count, b1, b2, &c1, &c2);
  for (int64_t i = 0; i < n; ++i) {
    double m1 = b1 * m[i] + (1.0 - b1) * g[i];
    double v1 = b2 * v[i] + (1.0 - b2) * g[i] * g[i];
    double mh = m1 / c1;
    double vh = v1 / c2;
    double s = sqrt(vh + eps_root);
    double d = s + eps;
    double u = -lr * mh / d;
    m_out[i] = m1;
    v_out[i] = v1;
    if (u_out) u_out[i] = u;
    p_out[i] = p[i] + u;
  }
}

/*
 * Vector-Jacobian product of oracle_adam_fwd (Sec. 2.3: the backward of the
 * fused optimizer), plain chain rule through the forward's own steps.
 * Cotangents: dP on p', dM on m', dV on v' (dM, dV may be NULL = zero).
 *   dL/dm' = Mt = dM - dP lr / (c1 d)
 *   dL/dv' = Vt = dV + dP lr m^ / (2 c2 s d^2)      (dP term := 0 if s == 0, R3)
 *   dp = dP
 *   dg = (1-b1) Mt + 2 (1-b2) g Vt
 *   dm = b1 Mt
 *   dv = b2 Vt
 * dp_out may be NULL (it is the identity on dP).
 */
void oracle_adam_bwd(int64_t n, const double* dP, const double* dM,
                     const double* dV, const double* g, const double* m,
                     const double* v, int64_t count, double lr, double b1,
                     double b2, double eps, double eps_root, double* dp_out,
                     double* dg_out, double* dm_out, double* dv_out) {
  double c1, c2;
  bias_corrections(count, b1, b2, &c1, &c2);
  for (int64_t i = 0; i < n; ++i) {
    double m1 = b1 * m[i] + (1.0 - b1) * g[i];
    double v1 = b2 * v[i] + (1.0 - b2) * g[i] * g[i];
    double mh = m1 / c1;
    double vh = v1 / c2;
    double s = sqrt(vh + eps_root);
    double d = s + eps;
    double dMi = dM ? dM[i] : 0.0;
    double dVi = dV ? dV[i] : 0.0;
    double Mt = dMi - dP[i] * lr / (c1 * d);
    double Vt = dVi;
    if (s > 0.0) Vt += dP[i] * lr * mh / (2.0 * c2 * s * d * d);
    if (dp_out) dp_out[i] = dP[i];
    dg_out[i] = (1.0 - b1) * Mt + 2.0 * (1.0 - b2) * g[i] * Vt;
    dm_out[i] = b1 * Mt;
    dv_out[i] = b2 * Vt;
  }
}

/*
 * Tolerance scales for the forward outputs: for each output, the sum of the
 * absolute values of the terms that make it up.  A result computed with
 * relative rounding error r per operation differs from the exact value by a
 * small multiple of r times this scale, whatever cancellation occurs.
 *   mag(m') = b1|m| + (1-b1)|g|
 *   mag(v') = b2|v| + (1-b2) g^2
 *   mag(u)  = lr mag(m') / (c1 d)
 *   mag(p') = |p| + mag(u)
 */
void oracle_adam_fwd_mag(int64_t n, const double* p, const double* g,
                         const double* m, const double* v, int64_t count,
                         double lr, double b1, double b2, double eps,
                         double eps_root, double* mag_p, double* mag_m,
                         double* mag_v, double* mag_u) {
  double c1, c2;
  bias_corrections(count, b1, b2, &c1, &c2);
  for (int64_t i = 0; i < n; ++i) {
    double v1 = b2 * v[i] + (1.0 - b2) * g[i] * g[i];
    double s = sqrt(v1 / c2 + eps_root);
    double d = s + eps;
    double am = b1 * fabs(m[i]) + (1.0 - b1) * fabs(g[i]);
    double av = b2 * fabs(v[i]) + (1.0 - b2) * g[i] * g[i];
    double au = fabs(lr) * am / (c1 * d);
    mag_m[i] = am;
    mag_v[i] = av;
    mag_u[i] = au;
    mag_p[i] = fabs(p[i]) + au;
  }
}

/*
 * Tolerance scales for the backward outputs.  For dg the scale is taken from
 * the algebraically reduced form of the same quantity, in which the g^2 terms
 * of the plain chain rule cancel exactly (substitute v^ = b2 v/c2 + b g^2 and
 * m^ = b1 m/c1 + a g, with a = (1-b1)/c1, b = (1-b2)/c2):
 *   dg = (1-b1) dM + 2(1-b2) g dV + dP lr N / (s d^2),
 *   N  = b b1 g m / c1 - a b2 v / c2 - a (eps_root + s eps);
 * at s == 0 the dP term is -dP lr a / d (reading R3).
 *   mag(dg) = (1-b1)|dM| + 2(1-b2)|g dV|
 *             + |dP| lr (b b1 |g m|/c1 + a b2 |v|/c2 + a (eps_root + s eps)) / (s d^2)
 *   mag(dm) = b1 (|dM| + |dP| lr / (c1 d))
 *   mag(dv) = b2 (|dV| + |dP| lr mag(m^) / (2 c2 s d^2)),  mag(m^) = mag(m')/c1
 * This is the reduced form written out only to size a tolerance; the values
 * themselves come from oracle_adam_bwd.
 */
void oracle_adam_bwd_mag(int64_t n, const double* dP, const double* dM,
                         const double* dV, const double* g, const double* m,
                         const double* v, int64_t count, double lr, double b1,
                         double b2, double eps, double eps_root,
                         double* mag_dg, double* mag_dm, double* mag_dv) {
  double c1, c2;
  bias_corrections(count, b1, b2, &c1, &c2);
  double a = (1.0 - b1) / c1;
  double b = (1.0 - b2) / c2;
  for (int64_t i = 0; i < n; ++i) {
    double v1 = b2 * v[i] + (1.0 - b2) * g[i] * g[i];
    double s = sqrt(v1 / c2 + eps_root);
    double d = s + eps;
    double adP = fabs(dP[i]);
    double adM = dM ? fabs(dM[i]) : 0.0;
    double adV = dV ? fabs(dV[i]) : 0.0;
    double amh = (b1 * fabs(m[i]) + (1.0 - b1) * fabs(g[i])) / c1;
    double t3, tv;
    if (s > 0.0) {
      double num = b * b1 * fabs(g[i] * m[i]) / c1 + a * b2 * fabs(v[i]) / c2 +
                   a * (eps_root + s * eps);
      t3 = adP * fabs(lr) * num / (s * d * d);
      tv = adP * fabs(lr) * amh / (2.0 * c2 * s * d * d);
    } else {
      t3 = adP * fabs(lr) * a / d;
      tv = 0.0;
    }
    mag_dg[i] = (1.0 - b1) * adM + 2.0 * (1.0 - b2) * fabs(g[i]) * adV + t3;
    mag_dm[i] = b1 * (adM + adP * fabs(lr) / (c1 * d));
    mag_dv[i] = b2 * (adV + tv);
  }
}

/*
 * K-step unrolled forward (Listing 1's inner loop with given gradients):
 *   for k = 1..K: (p_k, m_k, v_k) = step(p_{k-1}, g_k, m_{k-1}, v_{k-1},
 *                                        count0 + k - 1)
 * grads: K*n row-major (step k at grads + (k-1)*n).
 * m_traj, v_traj: (K+1)*n; entry 0 is a copy of m0 / v0, entry k is m_k / v_k.
 * p_out: p_K.
 */
void oracle_unrolled_fwd(int64_t K, int64_t n, const double* p0,
                         const double* grads, const double* m0,
                         const double* v0, int64_t count0, double lr,
                         double b1, double b2, double eps, double eps_root,
                         double* p_out, double* m_traj, double* v_traj) {
  memcpy(m_traj, m0, (size_t)n * sizeof(double));
  memcpy(v_traj, v0, (size_t)n * sizeof(double));
  memcpy(p_out, p0, (size_t)n * sizeof(double));
  for (int64_t k = 1; k <= K; ++k) {
    oracle_adam_fwd(n, p_out, grads + (k - 1) * n, m_traj + (k - 1) * n,
                    v_traj + (k - 1) * n, count0 + k - 1, lr, b1, b2, eps,
                    eps_root, p_out, m_traj + k * n, v_traj + k * n, NULL);
  }
}

/*
 * K-step unrolled backward: reverse-mode through the K steps of
 * oracle_unrolled_fwd, starting from the cotangent dpK of p_K and zero
 * cotangents of m_K, v_K.
 *   for k = K..1: (dP, dg_k, dM, dV) = vjp_k(dP, dM, dV)
 * Outputs: dp0 (= dpK, the params path is the identity), dg (K*n, step k at
 * dg + (k-1)*n), dm0, dv0.  Inputs m_traj/v_traj as written by the forward.
 */
void oracle_unrolled_bwd(int64_t K, int64_t n, const double* dpK,
                         const double* grads, const double* m_traj,
                         const double* v_traj, int64_t count0, double lr,
                         double b1, double b2, double eps, double eps_root,
                         double* dp0, double* dg, double* dm0, double* dv0) {
  memcpy(dp0, dpK, (size_t)n * sizeof(double));
  for (int64_t i = 0; i < n; ++i) {
    dm0[i] = 0.0;
    dv0[i] = 0.0;
  }
  for (int64_t k = K; k >= 1; --k) {
    /* dm0/dv0 hold the cotangents of m_k/v_k on entry, of m_{k-1}/v_{k-1}
       on exit; each element is read before it is written. */
    oracle_adam_bwd(n, dp0, dm0, dv0, grads + (k - 1) * n,
                    m_traj + (k - 1) * n, v_traj + (k - 1) * n,
                    count0 + k - 1, lr, b1, b2, eps, eps_root, dp0,
                    dg + (k - 1) * n, dm0, dv0);
  }
}

/*
 * Tree pack (flatten), by definition: for every segment j,
 *   flat[off_j + i] = leaf_j[i],  0 <= i < numel_j,
 * copied as bytes (elem_bytes per element), so every bit pattern survives.
 * offsets == NULL means dense: off_j = sum of numel over segments before j.
 */
void oracle_pack(int64_t nseg, const int64_t* numel, const int64_t* offsets,
                 int64_t elem_bytes, const void* const* leaves, void* flat) {
  int64_t run = 0;
  for (int64_t j = 0; j < nseg; ++j) {
    int64_t off = offsets ? offsets[j] : run;
    memcpy((char*)flat + off * elem_bytes, leaves[j],
           (size_t)(numel[j] * elem_bytes));
    run += numel[j];
  }
}

/* Tree unpack (unflatten), the mirror: leaf_j[i] = flat[off_j + i]. */
void oracle_unpack(int64_t nseg, const int64_t* numel, const int64_t* offsets,
                   int64_t elem_bytes, const void* flat, void* const* leaves) {
  int64_t run = 0;
  for (int64_t j = 0; j < nseg; ++j) {
    int64_t off = offsets ? offsets[j] : run;
    memcpy(leaves[j], (const char*)flat + off * elem_bytes,
           (size_t)(numel[j] * elem_bytes));
    run += numel[j];
  }
}

/* ---------------------------------------------------------------------------
 * The paper's other fused differentiable optimizers (Sec. 1, contribution
 * (2)(i): SGD, RMSProp, Adam).  It prints no formula for them either; these
 * are the textbook forms, as torch.optim implements them.
 *
 * SGD with momentum mu >= 0 (trace t, zero initially; mu = 0 is plain SGD):
 *   t' = mu t + g
 *   u  = -lr t'                (nesterov: u = -lr (g + mu t'))
 *   p' = p + u
 * t_out may be NULL when mu == 0 (no state).
 */
void oracle_sgd_fwd(int64_t n, const double* p, const double* g, const double* t, double lr, double mu,
                    int64_t nesterov, double* p_out, double* t_out) {
  for (int64_t i = 0; i < n; ++i) {
    double t1 = (t ? mu * t[i] : 0.0) + g[i];
    double u = nesterov ? -lr * (g[i] + mu * t1) : -lr * t1;
    if (t_out) t_out[i] = t1;
    p_out[i] = p[i] + u;
  }
}

/* VJP of oracle_sgd_fwd, chain rule.  Cotangents dP on p', dT on t' (NULL =
 * zero).  dL/dt' = dT - lr dP (nesterov: dT - lr mu dP);
 *   dg = dL/dt' (+ nesterov: - lr dP),  dt = mu dL/dt',  dp = dP.
 * The map is linear, so the VJP does not depend on p, g or t. */
void oracle_sgd_bwd(int64_t n, const double* dP, const double* dT, double lr, double mu, int64_t nesterov,
                    double* dg_out, double* dt_out) {
  for (int64_t i = 0; i < n; ++i) {
    double dTi = dT ? dT[i] : 0.0;
    double Tt = dTi - (nesterov ? lr * mu : lr) * dP[i];
    dg_out[i] = Tt - (nesterov ? lr * dP[i] : 0.0);
    if (dt_out) dt_out[i] = mu * Tt;
  }
}

/*
 * RMSProp with decay alpha in [0, 1), eps outside and eps_root inside the
 * root, optional momentum mu >= 0 (buffer b, zero initially):
 *   v' = alpha v + (1-alpha) g^2
 *   s  = sqrt(v' + eps_root),  d = s + eps
 *   mu == 0:  u = -lr g / d
 *   mu >  0:  b' = mu b + g / d,  u = -lr b'
 *   p' = p + u
 * b, b_out are unused (may be NULL) when mu == 0.
 */
void oracle_rmsprop_fwd(int64_t n, const double* p, const double* g, const double* v, const double* b, double lr,
                        double alpha, double eps, double eps_root, double mu, double* p_out, double* v_out,
                        double* b_out) {
  for (int64_t i = 0; i < n; ++i) {
    double v1 = alpha * v[i] + (1.0 - alpha) * g[i] * g[i];
    double s = sqrt(v1 + eps_root);
    double d = s + eps;
    double q = g[i] / d;
    double u;
    if (mu > 0.0) {
      double b1 = mu * (b ? b[i] : 0.0) + q;
      if (b_out) b_out[i] = b1;
      u = -lr * b1;
    } else {
      u = -lr * q;
    }
    v_out[i] = v1;
    p_out[i] = p[i] + u;
  }
}

/* VJP of oracle_rmsprop_fwd, plain chain rule.  Cotangents dP on p', dV on v',
 * dB on b' (dV, dB NULL = zero; dB unused when mu == 0).
 *   Bt = dB - lr dP            (mu > 0: cotangent of b');  mu == 0: Bt = -lr dP
 *   dL/d(g/d) = Bt
 *   Vt = dV - Bt g / (2 s d^2)   (the Bt term := 0 when s == 0, reading R3)
 *   dg = Bt / d + 2 (1-alpha) g Vt,  dv = alpha Vt,  db = mu Bt,  dp = dP
 * At s == 0 (eps_root = 0, v = 0, g = 0) this gives dg's Bt term Bt / eps,
 * the symmetric derivative of g / d at g = 0. */
void oracle_rmsprop_bwd(int64_t n, const double* dP, const double* dV, const double* dB, const double* g,
                        const double* v, double lr, double alpha, double eps, double eps_root, double mu,
                        double* dg_out, double* dv_out, double* db_out) {
  for (int64_t i = 0; i < n; ++i) {
    double v1 = alpha * v[i] + (1.0 - alpha) * g[i] * g[i];
    double s = sqrt(v1 + eps_root);
    double d = s + eps;
    double Bt = (mu > 0.0 ? (dB ? dB[i] : 0.0) : 0.0) - lr * dP[i];
    double Vt = dV ? dV[i] : 0.0;
    if (s > 0.0) Vt -= Bt * g[i] / (2.0 * s * d * d);
    dg_out[i] = Bt / d + 2.0 * (1.0 - alpha) * g[i] * Vt;
    dv_out[i] = alpha * Vt;
    if (db_out) db_out[i] = mu * Bt;
  }
}

/* Tolerance scales for RMSProp (sums of |terms|; for dg taken from the
 * algebraically reduced form dg = 2(1-alpha) g dV + Bt (alpha v + eps_root +
 * s eps) / (s d^2), in which the g^2 terms of the chain rule cancel). */
void oracle_rmsprop_fwd_mag(int64_t n, const double* p, const double* g, const double* v, const double* b,
                            double lr, double alpha, double eps, double eps_root, double mu, double* mag_p,
                            double* mag_v, double* mag_b) {
  for (int64_t i = 0; i < n; ++i) {
    double v1 = alpha * fabs(v[i]) + (1.0 - alpha) * g[i] * g[i];
    double s = sqrt(alpha * v[i] + (1.0 - alpha) * g[i] * g[i] + eps_root);
    double d = s + eps;
    double aq = fabs(g[i]) / d;
    double ab = mu > 0.0 ? mu * fabs(b ? b[i] : 0.0) + aq : aq;
    mag_v[i] = v1;
    if (mag_b) mag_b[i] = ab;
    mag_p[i] = fabs(p[i]) + fabs(lr) * ab;
  }
}

void oracle_rmsprop_bwd_mag(int64_t n, const double* dP, const double* dV, const double* dB, const double* g,
                            const double* v, double lr, double alpha, double eps, double eps_root, double mu,
                            double* mag_dg, double* mag_dv, double* mag_db) {
  for (int64_t i = 0; i < n; ++i) {
    double s = sqrt(alpha * v[i] + (1.0 - alpha) * g[i] * g[i] + eps_root);
    double d = s + eps;
    double aBt = (mu > 0.0 ? fabs(dB ? dB[i] : 0.0) : 0.0) + fabs(lr) * fabs(dP[i]);
    double adV = dV ? fabs(dV[i]) : 0.0;
    double t3 = s > 0.0 ? aBt * (alpha * fabs(v[i]) + eps_root + s * eps) / (s * d * d) : aBt / d;
    double tv = s > 0.0 ? aBt * fabs(g[i]) / (2.0 * s * d * d) : 0.0;
    mag_dg[i] = 2.0 * (1.0 - alpha) * fabs(g[i]) * adV + t3;
    mag_dv[i] = alpha * (adV + tv);
    if (mag_db) mag_db[i] = mu * aBt;
  }
}

/* ---------------------------------------------------------------------------
 * Zero-order (evolution-strategies) gradient estimation (Sec. 2.2 "Zero-order
 * Differentiation"): the gradient of the Gaussian smoothing
 * f_s(theta) = E_z[f(theta + s z)], z ~ N(0, I), is (1/s) E_z[f(theta + s z) z].
 * Monte-Carlo with N given noise vectors z_1..z_N (rows of `noise`, N x n):
 *
 * es_perturb: the points to evaluate, row i of out = theta + s z_i; with
 *   antithetic sampling also row N + i = theta - s z_i (out has 2N rows).
 */
void oracle_es_perturb(int64_t N, int64_t n, const double* theta, const double* noise, double sigma,
                       int64_t antithetic, double* out) {
  for (int64_t i = 0; i < N; ++i)
    for (int64_t j = 0; j < n; ++j) {
      out[i * n + j] = theta[j] + sigma * noise[i * n + j];
      if (antithetic) out[(N + i) * n + j] = theta[j] - sigma * noise[i * n + j];
    }
}

/* es_estimate: grad_j = scale * sum_i w_i z_ij, summed in sample order.  The
 * caller forms the weights from the evaluated values f_i:
 *   plain:       w_i = f(theta + s z_i),                         scale = 1/(N s)
 *   baseline:    w_i = f(theta + s z_i) - f(theta),              scale = 1/(N s)
 *   antithetic:  w_i = f(theta + s z_i) - f(theta - s z_i),      scale = 1/(2 N s) */
void oracle_es_estimate(int64_t N, int64_t n, const double* noise, const double* w, double scale, double* grad) {
  for (int64_t j = 0; j < n; ++j) {
    double acc = 0.0;
    for (int64_t i = 0; i < N; ++i) acc += w[i] * noise[i * n + j];
    grad[j] = scale * acc;
  }
}

/* ---------------------------------------------------------------------------
 * Gaussian noise for the zero-order estimator, drawn from a counter-based
 * generator so that every element z_ij (sample i, parameter j) is a pure
 * function of (seed, i, j): the noise never has to be stored, and either
 * side regenerates any element on its own.  Sec. 2.2 / Listing 3 make the
 * noise sampler part of the estimator; the paper names no generator, so this
 * is a reading (its published sources are named below).
 *
 * Philox-4x64-10 (Salmon, Moraes, Dror and Shaw, "Parallel random numbers:
 * as easy as 1, 2, 3", SC 2011): a 256-bit counter block c = (c0..c3) and a
 * 128-bit key k = (k0, k1) go through ten rounds; each round forms the full
 * 128-bit products M0 c0 = (hi0, lo0) and M1 c2 = (hi1, lo1) and maps
 *   c <- (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0),
 * and between rounds the key advances by the Weyl increments W0, W1
 * (wrapping).  The four words of the last round are the output block.
 */
#define PHILOX_M0 0xD2E7470EE14C6C93ull
#define PHILOX_M1 0xCA5A826395121157ull
#define PHILOX_W0 0x9E3779B97F4A7C15ull
#define PHILOX_W1 0xBB67AE8584CAA73Bull

void oracle_philox4x64_10(const uint64_t* ctr, const uint64_t* key, uint64_t* out) {
  uint64_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
  uint64_t k0 = key[0], k1 = key[1];
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += PHILOX_W0;
      k1 += PHILOX_W1;
    }
    unsigned __int128 p0 = (unsigned __int128)PHILOX_M0 * c0;
    unsigned __int128 p1 = (unsigned __int128)PHILOX_M1 * c2;
    uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
    uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
    uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  out[0] = c0;
  out[1] = c1;
  out[2] = c2;
  out[3] = c3;
}

/*
 * Box-Muller transform (Box and Muller, 1958) of one 64-bit word: its low
 * 32 bits give u1 = (floor(lo / 2^8) + 1) 2^-24 in (0, 1], its high 32 bits
 * u2 = floor(hi / 2^8) 2^-24 in [0, 1) (24-bit uniforms, exact in fp32 and
 * fp64), and
 *   r = sqrt(-2 ln u1),   za = r cos(2 pi u2),   zb = r sin(2 pi u2)
 * are two independent standard normal draws.
 */
void oracle_box_muller(uint64_t word, double* za, double* zb) {
  uint32_t lo = (uint32_t)word, hi = (uint32_t)(word >> 32);
  double u1 = ((double)(lo >> 8) + 1.0) * 0x1p-24;
  double u2 = (double)(hi >> 8) * 0x1p-24;
  double r = sqrt(-2.0 * log(u1));
  double a = 6.283185307179586476925 * u2; /* 2 pi, rounded to double */
  *za = r * cos(a);
  *zb = r * sin(a);
}

/*
 * Which parameters a Philox block covers.  The parameters are cut into
 * segments of 512; block c = 64 s + l (segment s, slot l < 64) covers the
 * four parameters 512 s + 4 l + e and the four parameters 512 s + 256 + 4 l + e
 * (e < 4): word 2 h + e / 2 of the block (h = 0 for the first four, 1 for the
 * second) gives parameters with even e its cosine normal and odd e its sine
 * normal.  (This puts the eight normals of one block into two 16-byte vectors
 * 1 KiB apart, so 64 consecutive blocks fill two contiguous 1 KiB runs.)
 * noise_slot maps a parameter index to its block, word and normal.
 */
static void noise_slot(int64_t j, uint64_t* block, int* word, int* odd) {
  int64_t s = j / 512, q = j % 512;
  *block = (uint64_t)(64 * s + (q % 256) / 4);
  *word = 2 * (int)(q / 256) + (int)(q % 4) / 2;
  *odd = (int)(q % 2);
}

/*
 * The noise matrix z (N x n, row-major) for a seed: element j of sample i is
 * the normal noise_slot(j) names in the Philox block at counter
 * (block, i, 0, 0) under key (seed, 0), through the Box-Muller transform.
 */
void oracle_es_gaussian_noise(int64_t N, int64_t n, uint64_t seed, double* z) {
  uint64_t key[2] = {seed, 0};
  int64_t nblocks = 64 * ((n + 511) / 512);
  for (int64_t i = 0; i < N; ++i)
    for (int64_t b = 0; b < nblocks; ++b) {
      uint64_t ctr[4] = {(uint64_t)b, (uint64_t)i, 0, 0}, out[4];
      oracle_philox4x64_10(ctr, key, out);
      for (int h = 0; h < 2; ++h)
        for (int e = 0; e < 4; ++e) {
          int64_t j = 512 * (b / 64) + 256 * h + 4 * (b % 64) + e;
          if (j >= n) continue;
          double za, zb;
          oracle_box_muller(out[2 * h + e / 2], &za, &zb);
          z[i * n + j] = (e % 2 == 0) ? za : zb;
        }
    }
}

/*
 * Weights and scale of the Monte-Carlo estimate from the caller's
 * evaluations f (reading 17 of the design notes):
 *   method 0, plain:      w_i = f_i,              scale = 1 / (N s)    (f has N values)
 *   method 1, baseline:   w_i = f_i - f0,         scale = 1 / (N s)    (f0 = f(theta))
 *   method 2, antithetic: w_i = f_i - f_{N+i},    scale = 1 / (2 N s)  (f has 2N values:
 *                         the points theta + s z_i, then theta - s z_i)
 * so that grad = scale * sum_i w_i z_i (oracle_es_estimate).
 */
void oracle_es_weights(int64_t N, const double* f, double f0, int64_t method, double sigma, double* w,
                       double* scale) {
  for (int64_t i = 0; i < N; ++i) {
    if (method == 0)
      w[i] = f[i];
    else if (method == 1)
      w[i] = f[i] - f0;
    else
      w[i] = f[i] - f[N + i];
  }
  *scale = 1.0 / ((method == 2 ? 2.0 : 1.0) * (double)N * sigma);
}

/* Tolerance scale of each noise element: the radius r = sqrt(-2 ln u1) of
 * its Box-Muller pair.  z = r cos(a) (or r sin(a)) is the product of r and a
 * factor of magnitude up to 1 whose rounding is absolute, so r, not |z|,
 * sizes the error of a computed z. */
void oracle_es_gaussian_noise_radius(int64_t N, int64_t n, uint64_t seed, double* r) {
  uint64_t key[2] = {seed, 0};
  for (int64_t i = 0; i < N; ++i)
    for (int64_t j = 0; j < n; ++j) {
      uint64_t block, out[4];
      int word, odd;
      noise_slot(j, &block, &word, &odd);
      uint64_t ctr[4] = {block, (uint64_t)i, 0, 0};
      oracle_philox4x64_10(ctr, key, out);
      uint32_t lo = (uint32_t)out[word];
      r[i * n + j] = sqrt(-2.0 * log(((double)(lo >> 8) + 1.0) * 0x1p-24));
    }
}

/* The same noise (and radius) at chosen parameters only: z[i * ncols + c] is
 * element cols[c] of sample i, by the definition above.  For sampled checks
 * of large estimates. */
void oracle_es_gaussian_noise_cols(int64_t N, int64_t ncols, const int64_t* cols, uint64_t seed, double* z,
                                   double* r) {
  uint64_t key[2] = {seed, 0};
  for (int64_t i = 0; i < N; ++i)
    for (int64_t c = 0; c < ncols; ++c) {
      uint64_t block, out[4];
      int word, odd;
      noise_slot(cols[c], &block, &word, &odd);
      uint64_t ctr[4] = {block, (uint64_t)i, 0, 0};
      oracle_philox4x64_10(ctr, key, out);
      double za, zb;
      oracle_box_muller(out[word], &za, &zb);
      z[i * ncols + c] = odd ? zb : za;
      uint32_t lo = (uint32_t)out[word];
      r[i * ncols + c] = sqrt(-2.0 * log(((double)(lo >> 8) + 1.0) * 0x1p-24));
    }
}
