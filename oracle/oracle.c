/*
 * oracle.c -- plain fp64 CPU oracle for the block-hybrid attention layer of
 * "Retrofitting Linear Attention into Diffusion Language Models".
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the library path may link, load or
 * call this file; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no source with the HIP library: every index
 * below is written from the documented buffer layouts, not from the kernels.
 *
 * Every quantity is evaluated in double precision, literally as the paper
 * defines it (no max-shift, no blocking, no reordering).  The only guard is
 * that a softmax exponent must stay below 700 in magnitude, so that exp()
 * cannot overflow a double; a call that would break it returns 1.
 *
 * Layouts (row-major, contiguous, indices outermost first):
 *   q, out        [B][L][Hq][d]      (prefill: [B][T][Hq][d])
 *   k, v          [B][L][Hkv][d]     (prefill: [B][T][Hkv][d])
 *   Wt            [Hq][F][d]         Wt[h][j][i] = W_h[i][j], W_h in R^{d x F}
 *   alpha         [Hq]               gate logit, w = sigmoid(alpha)
 *   S             [n_slots][Hq][2F][d]
 *   z             [n_slots][Hq][2F]
 *   slots         [B] or NULL        state slot of request b (NULL: slot b)
 *   k_cache,v_cache [B][Pmax][Hkv][d], request b uses its first plen[b] rows
 * Query head h reads KV head h / (Hq / Hkv).
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC oracle.c -o liboracle.so -lm
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Threads of the OpenMP loops below (the host-core count of a timing). */
void oracle_set_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }
int oracle_max_threads(void) { return omp_get_max_threads(); }

#define EXP_LIMIT 700.0

/* Feature map of Section 3.1 ("Across blocks"):
 *   phi(x) = [ softmax(x W), softmax(-x W) ]  in R^{2F},
 * with the softmax taken over the F entries of the row vector x W.
 * The paper fixes no stabilising shift; the literal exp is used and the
 * exponent is checked.  Returns 1 if |x W|_inf >= EXP_LIMIT. */
static int feature_map(const double *x, const double *Wt, int d, int F,
                       double *phi) {
  double *pos = phi, *neg = phi + F;
  double sum_pos = 0.0, sum_neg = 0.0;
  for (int j = 0; j < F; ++j) {
    double u = 0.0; /* (x W)_j = sum_i x_i W[i][j] */
    for (int i = 0; i < d; ++i) u += x[i] * Wt[(size_t)j * d + i];
    if (fabs(u) >= EXP_LIMIT) return 1;
    pos[j] = exp(u);
    neg[j] = exp(-u);
    sum_pos += pos[j];
    sum_neg += neg[j];
  }
  for (int j = 0; j < F; ++j) {
    pos[j] /= sum_pos;
    neg[j] /= sum_neg;
  }
  return 0;
}

/* w = sigma(alpha), the per-head gate of Section 3.1 ("Combining the two
 * branches"). */
static double gate(double alpha) { return 1.0 / (1.0 + exp(-alpha)); }

/* One query of the block-hybrid output (Section 3.1):
 *   a_j     = exp(q . k_j / sqrt(d))                   over the active block
 *   sm_num  = sum_j a_j v_j,    sm_den = sum_j a_j
 *   lin_num = phi(q)^T S,       lin_den = phi(q)^T Z
 *   out     = (w sm_num + lin_num) / (w sm_den + lin_den)
 * kblk/vblk point at the first block token; consecutive block tokens are
 * tok_stride doubles apart.  scratch holds 2F + d doubles. */
static int hybrid_query(const double *q, const double *kblk,
                        const double *vblk, size_t tok_stride, int L, int d,
                        int F, const double *Wt, double w, const double *S,
                        const double *z, double *scratch, double *out) {
  const int f = 2 * F;
  double *phi = scratch, *sm_num = scratch + f;
  double sm_den = 0.0;
  for (int c = 0; c < d; ++c) sm_num[c] = 0.0;
  for (int j = 0; j < L; ++j) {
    const double *kj = kblk + (size_t)j * tok_stride;
    const double *vj = vblk + (size_t)j * tok_stride;
    double s = 0.0;
    for (int i = 0; i < d; ++i) s += q[i] * kj[i];
    s /= sqrt((double)d);
    if (fabs(s) >= EXP_LIMIT) return 1;
    double a = exp(s);
    sm_den += a;
    for (int c = 0; c < d; ++c) sm_num[c] += a * vj[c];
  }
  if (feature_map(q, Wt, d, F, phi)) return 1;
  double lin_den = 0.0;
  for (int r = 0; r < f; ++r) lin_den += phi[r] * z[r];
  double den = w * sm_den + lin_den;
  for (int c = 0; c < d; ++c) {
    double lin_num = 0.0;
    for (int r = 0; r < f; ++r) lin_num += phi[r] * S[(size_t)r * d + c];
    out[c] = (w * sm_num[c] + lin_num) / den;
  }
  return 0;
}

/* Commit of one token (Section 3.1 state update):
 *   S += phi(k) v^T,   Z += phi(k). */
static int commit_token(const double *kt, const double *vt, int d, int F,
                        const double *Wt, double *S, double *z,
                        double *phi) {
  const int f = 2 * F;
  if (feature_map(kt, Wt, d, F, phi)) return 1;
  for (int r = 0; r < f; ++r) {
    z[r] += phi[r];
    for (int c = 0; c < d; ++c) S[(size_t)r * d + c] += phi[r] * vt[c];
  }
  return 0;
}

static int slot_of(const int32_t *slots, int b) { return slots ? slots[b] : b; }

/* hybrid step: every query of the active block of every request and head. */
int oracle_step(int B, int Hq, int Hkv, int d, int L, int F, const double *q,
                const double *k, const double *v, const double *Wt,
                const double *alpha, const double *S, const double *z,
                const int32_t *slots, double *out) {
  const int G = Hq / Hkv, f = 2 * F;
  int err = 0;
#pragma omp parallel for schedule(dynamic) reduction(| : err)
  for (long u = 0; u < (long)B * Hq; ++u) {
    const int b = (int)(u / Hq), h = (int)(u % Hq), g = h / G;
    const int slot = slot_of(slots, b);
    const double *Sh = S + ((size_t)slot * Hq + h) * f * d;
    const double *zh = z + ((size_t)slot * Hq + h) * f;
    const double *Wh = Wt + (size_t)h * F * d;
    const double w = gate(alpha[h]);
    double *scratch = (double *)malloc(sizeof(double) * (f + d));
    const double *kblk = k + ((size_t)b * L * Hkv + g) * d;
    const double *vblk = v + ((size_t)b * L * Hkv + g) * d;
    for (int i = 0; i < L; ++i) {
      const size_t qo = (((size_t)b * L + i) * Hq + h) * d;
      err |= hybrid_query(q + qo, kblk, vblk, (size_t)Hkv * d, L, d, F, Wh, w,
                          Sh, zh, scratch, out + qo);
    }
    free(scratch);
  }
  return err;
}

/* commit: fold every token of the given block into the state of its slot. */
int oracle_commit(int B, int Hq, int Hkv, int d, int L, int F, const double *k,
                  const double *v, const double *Wt, double *S, double *z,
                  const int32_t *slots) {
  const int G = Hq / Hkv, f = 2 * F;
  int err = 0;
#pragma omp parallel for schedule(dynamic) reduction(| : err)
  for (long u = 0; u < (long)B * Hq; ++u) {
    const int b = (int)(u / Hq), h = (int)(u % Hq), g = h / G;
    const int slot = slot_of(slots, b);
    double *Sh = S + ((size_t)slot * Hq + h) * f * d;
    double *zh = z + ((size_t)slot * Hq + h) * f;
    const double *Wh = Wt + (size_t)h * F * d;
    double *phi = (double *)malloc(sizeof(double) * f);
    for (int t = 0; t < L; ++t) {
      const size_t ko = (((size_t)b * L + t) * Hkv + g) * d;
      err |= commit_token(k + ko, v + ko, d, F, Wh, Sh, zh, phi);
    }
    free(phi);
  }
  return err;
}

/* prefill of T = nblk * L tokens with the block-causal pattern of Figure 2:
 * block c is first read against the state of blocks 0..c-1 (hybrid step),
 * then committed.  out may be NULL (state only); q is then unused.  The state
 * starts from whatever S, z hold, so a prefill continues an earlier one. */
int oracle_prefill(int B, int T, int Hq, int Hkv, int d, int L, int F,
                   const double *q, const double *k, const double *v,
                   const double *Wt, const double *alpha, double *S, double *z,
                   const int32_t *slots, double *out) {
  const int G = Hq / Hkv, f = 2 * F;
  if (L <= 0 || T % L != 0) return 2;
  const int nblk = T / L;
  int err = 0;
#pragma omp parallel for schedule(dynamic) reduction(| : err)
  for (long u = 0; u < (long)B * Hq; ++u) {
    const int b = (int)(u / Hq), h = (int)(u % Hq), g = h / G;
    const int slot = slot_of(slots, b);
    double *Sh = S + ((size_t)slot * Hq + h) * f * d;
    double *zh = z + ((size_t)slot * Hq + h) * f;
    const double *Wh = Wt + (size_t)h * F * d;
    const double w = gate(alpha[h]);
    double *scratch = (double *)malloc(sizeof(double) * (f + d));
    for (int c = 0; c < nblk; ++c) {
      const size_t t0 = (size_t)c * L;
      const double *kblk = k + (((size_t)b * T + t0) * Hkv + g) * d;
      const double *vblk = v + (((size_t)b * T + t0) * Hkv + g) * d;
      if (out) {
        for (int i = 0; i < L; ++i) {
          const size_t qo = (((size_t)b * T + t0 + i) * Hq + h) * d;
          err |= hybrid_query(q + qo, kblk, vblk, (size_t)Hkv * d, L, d, F,
                              Wh, w, Sh, zh, scratch, out + qo);
        }
      }
      for (int t = 0; t < L; ++t) {
        const size_t ko = (((size_t)b * T + t0 + t) * Hkv + g) * d;
        err |= commit_token(k + ko, v + ko, d, F, Wh, Sh, zh, scratch);
      }
    }
    free(scratch);
  }
  return err;
}

/* Exact softmax attention (Section 2.2 display, without the causal mask
 * inside the block) of every block query over the request's cached prefix
 * plus all L block keys:
 *   out_i = sum_j exp(s_ij) v_j / sum_j exp(s_ij),  s_ij = q_i . k_j / sqrt(d)
 * j runs over k_cache[b][0 .. plen[b]-1] followed by the block keys. */
int oracle_softmax_prefix(int B, int Hq, int Hkv, int d, int L, int Pmax,
                          const double *q, const double *k, const double *v,
                          const double *k_cache, const double *v_cache,
                          const int32_t *plen, double *out) {
  const int G = Hq / Hkv;
  int err = 0;
#pragma omp parallel for schedule(dynamic) reduction(| : err)
  for (long u = 0; u < (long)B * Hq * L; ++u) {
    const int i = (int)(u % L);
    const int h = (int)((u / L) % Hq), b = (int)(u / ((long)L * Hq));
    const int g = h / G, P = plen[b];
    const size_t qo = (((size_t)b * L + i) * Hq + h) * d;
    const double *qi = q + qo;
    double *acc = (double *)calloc((size_t)d, sizeof(double));
    double den = 0.0;
    for (int j = 0; j < P + L; ++j) {
      const double *kj, *vj;
      if (j < P) {
        const size_t o = (((size_t)b * Pmax + j) * Hkv + g) * d;
        kj = k_cache + o;
        vj = v_cache + o;
      } else {
        const size_t o = (((size_t)b * L + (j - P)) * Hkv + g) * d;
        kj = k + o;
        vj = v + o;
      }
      double s = 0.0;
      for (int t = 0; t < d; ++t) s += qi[t] * kj[t];
      s /= sqrt((double)d);
      if (fabs(s) >= EXP_LIMIT) err = 1;
      double a = exp(s);
      den += a;
      for (int c = 0; c < d; ++c) acc[c] += a * vj[c];
    }
    for (int c = 0; c < d; ++c) out[qo + c] = acc[c] / den;
    free(acc);
  }
  return err;
}

/* The feature map alone, for pinning it: X [n][d] -> PHI [n][2F]. */
int oracle_feature_map(int n, int d, int F, const double *X, const double *Wt,
                       double *PHI) {
  int err = 0;
  for (int t = 0; t < n; ++t)
    err |= feature_map(X + (size_t)t * d, Wt, d, F, PHI + (size_t)t * 2 * F);
  return err;
}

/* ---------------------------------------------------------------------------
 * Backward of the block-causal hybrid layer over a training sequence, for the
 * attention transfer of Section 3.2 (Stage 1): the trainable parameters are
 * psi = {W, alpha}, so the gradients returned are dL/dW and dL/dalpha.
 *
 * Forward (the prefill pattern of Figure 2, from an empty state): block c of
 * the T = nblk * L tokens is answered as in hybrid_query against S_{c-1},
 * z_{c-1} (the blocks before it), then committed.
 *
 * Objective.  With target == NULL, L = sum_i <dout_i, out_i> (so the result
 * is the vector-Jacobian product for an upstream gradient dout).  With a
 * target (the frozen softmax teacher's output a^sm of Section 3.2), L is the
 * attention-transfer loss sum_i |out_i - target_i|^2 and dout_i =
 * 2 (out_i - target_i); loss[h] receives its value per query head.
 *
 * Reverse mode, written from the definitions (N = w sm_num + lin_num,
 * D = w sm_den + lin_den, out = N / D, g = dL/dout):
 *   dL/dN_i      = g_i / D_i
 *   dL/dD_i      = -(g_i . out_i) / D_i
 *   dL/dw       += dL/dN_i . sm_num_i + dL/dD_i sm_den_i
 *   dL/dphi(q_i) = S_{c-1} dL/dN_i + z_{c-1} dL/dD_i          (i in block c)
 *   dL/dphi(k_t) = sum_{c' > c} sum_{i in c'} phi(q_i) (v_t . dL/dN_i + dL/dD_i)
 *                = G_c v_t + gz_c                              (t in block c)
 *     with G_c = sum_{c' > c} sum_{i in c'} phi(q_i) (dL/dN_i)^T, gz_c likewise
 *   feature map, u = x W (F entries), phi = [p, n], p = softmax(u),
 *   n = softmax(-u), dphi = [dp, dn]:
 *     dL/du_j = p_j (dp_j - <dp, p>) - n_j (dn_j - <dn, n>)
 *     dL/dW[:, j] += x dL/du_j         (x = q_i or k_t, head h's W)
 *   dL/dalpha = dL/dw * w (1 - w).
 * Outputs are sums over the batch: dWt [Hq][F][d] (same layout as Wt),
 * dalpha [Hq], loss [Hq] (may be NULL without a target).
 *
 * Gradients with respect to the layer's inputs q, k, v (what end-to-end
 * training through the hybrid layers needs, Stage 2 of Section 3.2), written
 * from the same definitions; a_ij = exp(s_ij), s_ij = q_i . k_j / sqrt(d) for
 * i, j in one block:
 *   softmax branch (d sm_num_i = w dL/dN_i, d sm_den_i = w dL/dD_i):
 *     dL/da_ij = w (dL/dN_i . v_j + dL/dD_i),   dL/ds_ij = a_ij dL/da_ij
 *     dL/dq_i += sum_j dL/ds_ij k_j / sqrt(d)
 *     dL/dk_j += sum_i dL/ds_ij q_i / sqrt(d)
 *     dL/dv_j += sum_i a_ij w dL/dN_i
 *   feature maps: dL/dx += W_h dL/du (x = q_i or k_t, as above)
 *   state: dL/dv_t += G_c^T phi(k_t)                           (t in block c)
 * dq [B][T][Hq][d]; dk, dv [B][T][Hkv][d], each summed over the query heads
 * that share the KV head (in head order).  Any of them may be NULL.
 * --------------------------------------------------------------------------- */

/* dL/du of the feature map at x (phi already evaluated there), added into
 * dWt as x dL/du_j, and (dx not NULL) into dx as W dL/du, i.e.
 * dx_i += sum_j W[i][j] dL/du_j with W[i][j] = Wt[j][i]. */
static void feature_map_backward(const double *x, const double *phi,
                                 const double *dphi, int d, int F,
                                 const double *Wt, double *dWt, double *dx) {
  const double *p = phi, *n = phi + F, *dp = dphi, *dn = dphi + F;
  double sp = 0.0, sn = 0.0;
  for (int j = 0; j < F; ++j) {
    sp += dp[j] * p[j];
    sn += dn[j] * n[j];
  }
  for (int j = 0; j < F; ++j) {
    const double du = p[j] * (dp[j] - sp) - n[j] * (dn[j] - sn);
    for (int i = 0; i < d; ++i) dWt[(size_t)j * d + i] += du * x[i];
    if (dx)
      for (int i = 0; i < d; ++i) dx[i] += Wt[(size_t)j * d + i] * du;
  }
}

int oracle_backward(int B, int T, int Hq, int Hkv, int d, int L, int F,
                    const double *q, const double *k, const double *v,
                    const double *Wt, const double *alpha, const double *dout,
                    const double *target, double *dWt, double *dalpha,
                    double *loss, double *dq, double *dk, double *dv) {
  const int G = Hq / Hkv, f = 2 * F;
  if (L <= 0 || T % L != 0) return 2;
  if ((dout == NULL) == (target == NULL)) return 2;
  const int nblk = T / L;
  const long units = (long)B * Hq;
  const double rs = 1.0 / sqrt((double)d);
  /* per-unit results, summed over the batch in a fixed order afterwards */
  double *u_dW = (double *)calloc((size_t)units * F * d, sizeof(double));
  double *u_dw = (double *)calloc((size_t)units, sizeof(double));
  double *u_loss = (double *)calloc((size_t)units, sizeof(double));
  /* per-unit dk, dv [units][T][d], summed over the heads of a group after */
  double *u_dk = dk ? (double *)calloc((size_t)units * T * d, sizeof(double)) : NULL;
  double *u_dv = dv ? (double *)calloc((size_t)units * T * d, sizeof(double)) : NULL;
  if (dq) memset(dq, 0, sizeof(double) * (size_t)B * T * Hq * d);
  int err = 0;
#pragma omp parallel for schedule(dynamic) reduction(| : err)
  for (long u = 0; u < units; ++u) {
    const int b = (int)(u / Hq), h = (int)(u % Hq), g = h / G;
    const double *Wh = Wt + (size_t)h * F * d;
    const double w = gate(alpha[h]);
    double *dWu = u_dW + (size_t)u * F * d;
    /* forward state, then the per-query adjoints kept for the reverse pass */
    double *S = (double *)calloc((size_t)f * d, sizeof(double));
    double *z = (double *)calloc((size_t)f, sizeof(double));
    double *phiq = (double *)malloc(sizeof(double) * (size_t)T * f);
    double *dN = (double *)malloc(sizeof(double) * (size_t)T * d);
    double *dD = (double *)malloc(sizeof(double) * (size_t)T);
    double *phi = (double *)malloc(sizeof(double) * f);
    double *dphi = (double *)malloc(sizeof(double) * f);
    double *sm_num = (double *)malloc(sizeof(double) * d);
    double *o = (double *)malloc(sizeof(double) * d);
    double *gi = (double *)malloc(sizeof(double) * d);
    double *dku = u_dk ? u_dk + (size_t)u * T * d : NULL;
    double *dvu = u_dv ? u_dv + (size_t)u * T * d : NULL;
    double dw = 0.0, ls = 0.0;
    for (int c = 0; c < nblk && !err; ++c) {
      const size_t t0 = (size_t)c * L;
      for (int i = 0; i < L; ++i) {
        const size_t qo = (((size_t)b * T + t0 + i) * Hq + h) * d;
        const double *qi = q + qo;
        /* the forward quantities of Section 3.1 for query i */
        double sm_den = 0.0;
        for (int cc = 0; cc < d; ++cc) sm_num[cc] = 0.0;
        for (int j = 0; j < L; ++j) {
          const size_t ko = (((size_t)b * T + t0 + j) * Hkv + g) * d;
          double s = 0.0;
          for (int x = 0; x < d; ++x) s += qi[x] * k[ko + x];
          s /= sqrt((double)d);
          if (fabs(s) >= EXP_LIMIT) err = 1;
          const double a = exp(s);
          sm_den += a;
          for (int cc = 0; cc < d; ++cc) sm_num[cc] += a * v[ko + cc];
        }
        double *ph = phiq + (size_t)(t0 + i) * f;
        if (feature_map(qi, Wh, d, F, ph)) err = 1;
        double lin_den = 0.0;
        for (int r = 0; r < f; ++r) lin_den += ph[r] * z[r];
        const double D = w * sm_den + lin_den;
        for (int cc = 0; cc < d; ++cc) {
          double lin_num = 0.0;
          for (int r = 0; r < f; ++r) lin_num += ph[r] * S[(size_t)r * d + cc];
          o[cc] = (w * sm_num[cc] + lin_num) / D;
        }
        /* upstream gradient */
        for (int cc = 0; cc < d; ++cc) {
          if (target) {
            const double e = o[cc] - target[qo + cc];
            ls += e * e;
            gi[cc] = 2.0 * e;
          } else {
            gi[cc] = dout[qo + cc];
          }
        }
        double go = 0.0;
        for (int cc = 0; cc < d; ++cc) go += gi[cc] * o[cc];
        double *dNi = dN + (size_t)(t0 + i) * d;
        const double dDi = -go / D;
        dD[t0 + i] = dDi;
        for (int cc = 0; cc < d; ++cc) dNi[cc] = gi[cc] / D;
        for (int cc = 0; cc < d; ++cc) dw += dNi[cc] * sm_num[cc];
        dw += dDi * sm_den;
        /* dL/dphi(q_i) against the state this block read */
        for (int r = 0; r < f; ++r) {
          double s = z[r] * dDi;
          for (int cc = 0; cc < d; ++cc) s += S[(size_t)r * d + cc] * dNi[cc];
          dphi[r] = s;
        }
        double *dqi = dq ? dq + qo : NULL;
        feature_map_backward(qi, ph, dphi, d, F, Wh, dWu, dqi);
        /* the block softmax branch: scores against every key of the block */
        if (dq || dku || dvu) {
          for (int j = 0; j < L; ++j) {
            const size_t ko = (((size_t)b * T + t0 + j) * Hkv + g) * d;
            double s = 0.0;
            for (int x = 0; x < d; ++x) s += qi[x] * k[ko + x];
            const double a = exp(s * rs);
            double da = dDi;
            for (int cc = 0; cc < d; ++cc) da += dNi[cc] * v[ko + cc];
            const double ds = a * w * da;
            if (dqi)
              for (int x = 0; x < d; ++x) dqi[x] += ds * k[ko + x] * rs;
            if (dku) {
              double *dkj = dku + (size_t)(t0 + j) * d;
              for (int x = 0; x < d; ++x) dkj[x] += ds * qi[x] * rs;
            }
            if (dvu) {
              double *dvj = dvu + (size_t)(t0 + j) * d;
              for (int cc = 0; cc < d; ++cc) dvj[cc] += a * w * dNi[cc];
            }
          }
        }
      }
      for (int t = 0; t < L; ++t) {
        const size_t ko = (((size_t)b * T + t0 + t) * Hkv + g) * d;
        err |= commit_token(k + ko, v + ko, d, F, Wh, S, z, phi);
      }
    }
    /* reverse pass over the blocks: G_c, gz_c hold the later blocks' sums */
    double *Gs = S, *gz = z; /* the forward state is no longer needed */
    memset(Gs, 0, sizeof(double) * (size_t)f * d);
    memset(gz, 0, sizeof(double) * (size_t)f);
    for (int c = nblk - 1; c >= 0 && !err; --c) {
      const size_t t0 = (size_t)c * L;
      for (int t = 0; t < L; ++t) {
        const size_t ko = (((size_t)b * T + t0 + t) * Hkv + g) * d;
        if (feature_map(k + ko, Wh, d, F, phi)) err = 1;
        for (int r = 0; r < f; ++r) {
          double s = gz[r];
          for (int cc = 0; cc < d; ++cc) s += Gs[(size_t)r * d + cc] * v[ko + cc];
          dphi[r] = s;
        }
        feature_map_backward(k + ko, phi, dphi, d, F, Wh,
                             dWu, dku ? dku + (size_t)(t0 + t) * d : NULL);
        if (dvu) {
          /* the state read by the later blocks: G_c^T phi(k_t) */
          double *dvt = dvu + (size_t)(t0 + t) * d;
          for (int cc = 0; cc < d; ++cc) {
            double s = 0.0;
            for (int r = 0; r < f; ++r) s += Gs[(size_t)r * d + cc] * phi[r];
            dvt[cc] += s;
          }
        }
      }
      for (int i = 0; i < L; ++i) {
        const double *ph = phiq + (size_t)(t0 + i) * f;
        const double *dNi = dN + (size_t)(t0 + i) * d;
        for (int r = 0; r < f; ++r) {
          gz[r] += ph[r] * dD[t0 + i];
          for (int cc = 0; cc < d; ++cc) Gs[(size_t)r * d + cc] += ph[r] * dNi[cc];
        }
      }
    }
    u_dw[u] = dw * w * (1.0 - w);
    u_loss[u] = ls;
    free(S); free(z); free(phiq); free(dN); free(dD); free(phi); free(dphi);
    free(sm_num); free(o); free(gi);
  }
  for (int h = 0; h < Hq; ++h) {
    double *dW = dWt + (size_t)h * F * d;
    memset(dW, 0, sizeof(double) * (size_t)F * d);
    dalpha[h] = 0.0;
    if (loss) loss[h] = 0.0;
    for (int b = 0; b < B; ++b) {
      const long u = (long)b * Hq + h;
      for (size_t x = 0; x < (size_t)F * d; ++x) dW[x] += u_dW[(size_t)u * F * d + x];
      dalpha[h] += u_dw[u];
      if (loss) loss[h] += u_loss[u];
    }
  }
  /* dk, dv: sum over the G query heads of each KV head, in head order */
  for (int pass = 0; pass < 2; ++pass) {
    double *dst = pass == 0 ? dk : dv;
    const double *src = pass == 0 ? u_dk : u_dv;
    if (!dst) continue;
    for (int b = 0; b < B; ++b)
      for (int t = 0; t < T; ++t)
        for (int g = 0; g < Hkv; ++g) {
          double *o = dst + (((size_t)b * T + t) * Hkv + g) * d;
          for (int x = 0; x < d; ++x) o[x] = 0.0;
          for (int h = g * G; h < (g + 1) * G; ++h) {
            const double *p = src + (((size_t)b * Hq + h) * T + t) * d;
            for (int x = 0; x < d; ++x) o[x] += p[x];
          }
        }
  }
  free(u_dW); free(u_dw); free(u_loss); free(u_dk); free(u_dv);
  return err;
}
