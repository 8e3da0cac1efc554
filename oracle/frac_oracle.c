/*
 * frac_oracle.c -- float64 CPU oracle for the Frac selective mode-bank scan.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, includes or
 * calls this file; only the test-suite, the smoke check and the CPU-baseline leg
 * of the benchmark load it.  It shares no code, header, table or constant with
 * the HIP path.
 *
 * What it computes ("Fractional State Space Transition for Long Sequence
 * Modeling", Sec. 3.2 and Appendix D, Algorithm "Frac state transition"):
 *
 *   per token t, head h (controls frozen over the step):
 *     effective step     dtt   = dt * lambda^(1/alpha)            (eq. tau-eff,
 *                                                                    eq. rho-beta-def-frac)
 *     retention          rho_m = exp(-dtt / tau_m)                (eq. rho-beta-def-frac)
 *     injection          beta_m = 1 - rho_m                       (Algorithm, step 3, and the
 *                                                                    remark after it: all experiments
 *                                                                    drop the 1/lambda factor)
 *     read weights       c  = softmax_m(-alpha ln tau_m + read_logit_m)   (eq. read-softmax)
 *     write weights      w  = softmax_m(-alpha ln tau_m + write_logit_m)  (same form, Sec. 3.2)
 *     write gains        kappa_m = beta_m * w_m                   (eq. frac-selective-update)
 *     state update       S_m <- rho_m S_m + kappa_m * B_t x_t^T   (eq. frac-selective-update,
 *                                                                    state of each mode widened
 *                                                                    to N x P by the B/C
 *                                                                    projections)
 *     readout            y_t = sum_m c_m S_m^T C_t + D_h x_t      (eq. frac-readout; direct
 *                                                                    feedthrough D of Sec. 3.3)
 *
 * The readout uses the state after this token's update (eq. frac-readout reads
 * s_{t,m}).  One independent problem per (batch, head); B and C are shared by the
 * heads of a group, g(h) = h * G / H.
 *
 * The backward pass is reverse-mode differentiation of exactly that loop, with
 * the state checkpointed every CKPT steps and recomputed inside each segment.
 * Everything is float64 and evaluated in the order written; the build uses no
 * fast-math flags.  Parallelism is OpenMP over independent (batch, head) pairs;
 * reductions over heads (dB, dC, dD) are done afterwards in a fixed order, so the
 * result does not depend on the thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define CKPT 64

typedef struct {
  int64_t batch, seqlen, nheads, headdim, dstate, ngroups, nmodes;
} frac_oracle_dims;

/* All arrays are host float64, C-contiguous.
 *   x [B,L,H,P]; dt, alpha [B,L,H]; lambda [B,L,H] or NULL (lambda = 1);
 *   Bm, Cm [B,L,G,N]; read_logit, write_logit [B,L,H,M] or NULL (zero logits);
 *   tau [M]; D [H] or NULL; init_state [B,H,M,N,P] or NULL (zero state). */
typedef struct {
  const double *x, *dt, *alpha, *lambda, *Bm, *Cm, *read_logit, *write_logit, *tau, *D, *init_state;
} frac_oracle_inputs;

/* Per-token coefficients of the mode bank. */
typedef struct {
  double s;       /* lambda^(1/alpha) */
  double dtt;     /* effective step */
  double *rho, *beta, *c, *w, *kappa;
} tok_coef;

static void softmax(int M, const double *z, double *out) {
  double mx = z[0];
  for (int m = 1; m < M; ++m) if (z[m] > mx) mx = z[m];
  double sum = 0.0;
  for (int m = 0; m < M; ++m) { out[m] = exp(z[m] - mx); sum += out[m]; }
  for (int m = 0; m < M; ++m) out[m] /= sum;
}

static void token_coefficients(int M, const double *tau, double dt, double alpha, double lam,
                               const double *rl, const double *wl, double *zbuf, tok_coef *k) {
  k->s = pow(lam, 1.0 / alpha);
  k->dtt = dt * k->s;
  for (int m = 0; m < M; ++m) {
    double z = -k->dtt / tau[m];
    k->rho[m] = exp(z);
    k->beta[m] = -expm1(z);
  }
  for (int m = 0; m < M; ++m) zbuf[m] = -alpha * log(tau[m]) + (rl ? rl[m] : 0.0);
  softmax(M, zbuf, k->c);
  for (int m = 0; m < M; ++m) zbuf[m] = -alpha * log(tau[m]) + (wl ? wl[m] : 0.0);
  softmax(M, zbuf, k->w);
  for (int m = 0; m < M; ++m) k->kappa[m] = k->beta[m] * k->w[m];
}

/* Geometric bank tau_m = tau_min * (tau_max/tau_min)^((m-1)/(M-1)), endpoints
 * included; M = 1 gives tau_min.  (Appendix E: geometric base timescales between
 * tau_min = 1 and tau_max = 2^17.) */
void frac_oracle_default_tau(int M, double tau_min, double tau_max, double *out) {
  if (M == 1) { out[0] = tau_min; return; }
  for (int m = 0; m < M; ++m)
    out[m] = tau_min * pow(tau_max / tau_min, (double)m / (double)(M - 1));
}

int frac_oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

static int check_dims(const frac_oracle_dims *d) {
  if (!d) return -1;
  if (d->batch < 0 || d->seqlen < 0 || d->nheads <= 0 || d->headdim <= 0 || d->dstate <= 0 ||
      d->ngroups <= 0 || d->nmodes <= 0)
    return -1;
  if (d->nheads % d->ngroups) return -1;
  return 0;
}

/* ------------------------------------------------------------------ forward */

int frac_oracle_forward(const frac_oracle_dims *d, const frac_oracle_inputs *in, double *y,
                        double *final_state) {
  if (check_dims(d) || !in || !in->x || !in->dt || !in->alpha || !in->Bm || !in->Cm || !in->tau || !y)
    return -1;
  const int64_t Bsz = d->batch, L = d->seqlen, H = d->nheads, P = d->headdim, N = d->dstate,
                G = d->ngroups;
  const int M = (int)d->nmodes;
  const int64_t MNP = (int64_t)M * N * P;

#pragma omp parallel
  {
    double *S = (double *)malloc(sizeof(double) * MNP);
    double *scratch = (double *)malloc(sizeof(double) * 6 * M);
    tok_coef k = {0, 0, scratch, scratch + M, scratch + 2 * M, scratch + 3 * M, scratch + 4 * M};
    double *zbuf = scratch + 5 * M;

#pragma omp for schedule(dynamic)
    for (int64_t bh = 0; bh < Bsz * H; ++bh) {
      const int64_t b = bh / H, h = bh % H, g = h * G / H;
      if (in->init_state) memcpy(S, in->init_state + bh * MNP, sizeof(double) * MNP);
      else memset(S, 0, sizeof(double) * MNP);
      const double Dh = in->D ? in->D[h] : 0.0;
      for (int64_t t = 0; t < L; ++t) {
        const int64_t ith = (b * L + t) * H + h;
        const double *xt = in->x + ith * P;
        const double *Bt = in->Bm + ((b * L + t) * G + g) * N;
        const double *Ct = in->Cm + ((b * L + t) * G + g) * N;
        token_coefficients(M, in->tau, in->dt[ith], in->alpha[ith], in->lambda ? in->lambda[ith] : 1.0,
                           in->read_logit ? in->read_logit + ith * M : NULL,
                           in->write_logit ? in->write_logit + ith * M : NULL, zbuf, &k);
        double *yt = y + ith * P;
        for (int64_t p = 0; p < P; ++p) yt[p] = Dh * xt[p];
        for (int m = 0; m < M; ++m) {
          double *Sm = S + (int64_t)m * N * P;
          for (int64_t n = 0; n < N; ++n) {
            double *row = Sm + n * P;
            const double kb = k.kappa[m] * Bt[n];
            for (int64_t p = 0; p < P; ++p) row[p] = k.rho[m] * row[p] + kb * xt[p];
            const double cc = k.c[m] * Ct[n];
            for (int64_t p = 0; p < P; ++p) yt[p] += cc * row[p];
          }
        }
      }
      if (final_state) memcpy(final_state + bh * MNP, S, sizeof(double) * MNP);
    }
    free(S);
    free(scratch);
  }
  return 0;
}

/* ----------------------------------------------------------------- backward */

/* Gradient outputs (host float64, caller-allocated, overwritten):
 *   dx [B,L,H,P], ddt [B,L,H], dBm, dCm [B,L,G,N] (summed over the heads of a group),
 *   dalpha [B,L,H], dlambda [B,L,H] (ignored when lambda is NULL),
 *   dread_logit, dwrite_logit [B,L,H,M], dD [H], dinit_state [B,H,M,N,P].
 * Any output pointer except dx may be NULL to skip it.  dy is required;
 * d_final_state [B,H,M,N,P] may be NULL (zero). */
typedef struct {
  double *dx, *ddt, *dBm, *dCm, *dalpha, *dlambda, *dread_logit, *dwrite_logit, *dD, *dinit_state;
} frac_oracle_grads;

int frac_oracle_backward(const frac_oracle_dims *d, const frac_oracle_inputs *in, const double *dy,
                         const double *d_final_state, frac_oracle_grads *out) {
  if (check_dims(d) || !in || !in->x || !in->dt || !in->alpha || !in->Bm || !in->Cm || !in->tau || !dy ||
      !out || !out->dx)
    return -1;
  const int64_t Bsz = d->batch, L = d->seqlen, H = d->nheads, P = d->headdim, N = d->dstate,
                G = d->ngroups;
  const int M = (int)d->nmodes;
  const int64_t MNP = (int64_t)M * N * P;
  const int64_t nseg = (L + CKPT - 1) / CKPT;
  const int64_t BH = Bsz * H;

  /* Per-(b,h) partial dB, dC and dD, reduced over heads afterwards in a fixed order. */
  double *dB_part = (double *)calloc((size_t)(BH * L * N > 0 ? BH * L * N : 1), sizeof(double));
  double *dC_part = (double *)calloc((size_t)(BH * L * N > 0 ? BH * L * N : 1), sizeof(double));
  double *dD_part = (double *)calloc((size_t)(BH > 0 ? BH : 1), sizeof(double));
  if (!dB_part || !dC_part || !dD_part) { free(dB_part); free(dC_part); free(dD_part); return -2; }

  int status = 0;
#pragma omp parallel
  {
    double *ckpt = (double *)malloc(sizeof(double) * (size_t)(nseg > 0 ? nseg : 1) * MNP);
    double *buf = (double *)malloc(sizeof(double) * CKPT * MNP);
    double *Gs = (double *)malloc(sizeof(double) * MNP);
    double *scratch = (double *)malloc(sizeof(double) * 16 * M);
    if (!ckpt || !buf || !Gs || !scratch) {
#pragma omp atomic write
      status = -2;
    }
    tok_coef k = {0, 0, scratch, scratch + M, scratch + 2 * M, scratch + 3 * M, scratch + 4 * M};
    double *zbuf = scratch + 5 * M;
    double *dc = scratch + 6 * M, *dkap = scratch + 7 * M, *drho = scratch + 8 * M;
    double *dbeta = scratch + 9 * M, *dw = scratch + 10 * M, *dzc = scratch + 11 * M,
           *dzw = scratch + 12 * M;

#pragma omp for schedule(dynamic)
    for (int64_t bh = 0; bh < BH; ++bh) {
      if (status) continue;
      const int64_t b = bh / H, h = bh % H, g = h * G / H;
      const double Dh = in->D ? in->D[h] : 0.0;
#define TOK(t) ((b * L + (t)) * H + h)
#define COEF(t)                                                                                         \
  token_coefficients(M, in->tau, in->dt[TOK(t)], in->alpha[TOK(t)], in->lambda ? in->lambda[TOK(t)] : 1.0, \
                     in->read_logit ? in->read_logit + TOK(t) * M : NULL,                               \
                     in->write_logit ? in->write_logit + TOK(t) * M : NULL, zbuf, &k)
      /* forward sweep: ckpt[s] = state entering segment s */
      double *S = buf; /* reuse buf[0] as running state for the sweep */
      if (in->init_state) memcpy(S, in->init_state + bh * MNP, sizeof(double) * MNP);
      else memset(S, 0, sizeof(double) * MNP);
      for (int64_t t = 0; t < L; ++t) {
        if (t % CKPT == 0) memcpy(ckpt + (t / CKPT) * MNP, S, sizeof(double) * MNP);
        COEF(t);
        const double *xt = in->x + TOK(t) * P;
        const double *Bt = in->Bm + ((b * L + t) * G + g) * N;
        for (int m = 0; m < M; ++m)
          for (int64_t n = 0; n < N; ++n) {
            double *row = S + ((int64_t)m * N + n) * P;
            const double kb = k.kappa[m] * Bt[n];
            for (int64_t p = 0; p < P; ++p) row[p] = k.rho[m] * row[p] + kb * xt[p];
          }
      }
      /* adjoint of the state, seeded by the gradient of the final state */
      if (d_final_state) memcpy(Gs, d_final_state + bh * MNP, sizeof(double) * MNP);
      else memset(Gs, 0, sizeof(double) * MNP);
      double dD_acc = 0.0;

      for (int64_t s = nseg - 1; s >= 0; --s) {
        const int64_t t0 = s * CKPT, t1 = (t0 + CKPT < L) ? t0 + CKPT : L;
        /* recompute S_t for t in [t0, t1): buf[j] = S_{t0+j} */
        for (int64_t t = t0; t < t1; ++t) {
          const double *prev = (t == t0) ? ckpt + s * MNP : buf + (t - t0 - 1) * MNP;
          double *cur = buf + (t - t0) * MNP;
          COEF(t);
          const double *xt = in->x + TOK(t) * P;
          const double *Bt = in->Bm + ((b * L + t) * G + g) * N;
          for (int m = 0; m < M; ++m)
            for (int64_t n = 0; n < N; ++n) {
              const int64_t o = ((int64_t)m * N + n) * P;
              const double kb = k.kappa[m] * Bt[n];
              for (int64_t p = 0; p < P; ++p) cur[o + p] = k.rho[m] * prev[o + p] + kb * xt[p];
            }
        }
        for (int64_t t = t1 - 1; t >= t0; --t) {
          const double *St = buf + (t - t0) * MNP;
          const double *Sp = (t == t0) ? ckpt + s * MNP : buf + (t - t0 - 1) * MNP;
          COEF(t);
          const int64_t ith = TOK(t);
          const double *xt = in->x + ith * P;
          const double *dyt = dy + ith * P;
          const double *Bt = in->Bm + ((b * L + t) * G + g) * N;
          const double *Ct = in->Cm + ((b * L + t) * G + g) * N;
          double *dBt = dB_part + (bh * L + t) * N;
          double *dCt = dC_part + (bh * L + t) * N;
          double *dxt = out->dx + ith * P;

          /* readout y_t = sum_m c_m S_{t,m}^T C_t + D x_t */
          for (int64_t p = 0; p < P; ++p) { dD_acc += dyt[p] * xt[p]; dxt[p] = Dh * dyt[p]; }
          for (int m = 0; m < M; ++m) {
            double acc = 0.0;
            for (int64_t n = 0; n < N; ++n) {
              const double *row = St + ((int64_t)m * N + n) * P;
              double sd = 0.0;
              for (int64_t p = 0; p < P; ++p) sd += row[p] * dyt[p];
              acc += Ct[n] * sd;                /* dc_m  = C^T S_m dy   */
              dCt[n] += k.c[m] * sd;            /* dC   += c_m S_m dy   */
            }
            dc[m] = acc;
            for (int64_t n = 0; n < N; ++n) { /* adjoint of S_t gets c_m C dy^T */
              double *grow = Gs + ((int64_t)m * N + n) * P;
              const double cc = k.c[m] * Ct[n];
              for (int64_t p = 0; p < P; ++p) grow[p] += cc * dyt[p];
            }
          }
          /* update S_t = rho S_{t-1} + kappa B x^T */
          for (int m = 0; m < M; ++m) {
            double dk = 0.0, dr = 0.0;
            for (int64_t n = 0; n < N; ++n) {
              const double *grow = Gs + ((int64_t)m * N + n) * P;
              const double *prow = Sp + ((int64_t)m * N + n) * P;
              double gx = 0.0, gs = 0.0;
              for (int64_t p = 0; p < P; ++p) {
                gx += grow[p] * xt[p];
                gs += grow[p] * prow[p];
                dxt[p] += k.kappa[m] * Bt[n] * grow[p];
              }
              dBt[n] += k.kappa[m] * gx;
              dk += Bt[n] * gx;
              dr += gs;
            }
            dkap[m] = dk;
            drho[m] = dr;
          }
          for (int m = 0; m < M; ++m) {
            double *Gm = Gs + (int64_t)m * N * P;
            for (int64_t i = 0; i < N * P; ++i) Gm[i] *= k.rho[m];
          }
          /* scalar chain: kappa = beta w; rho = exp(-dtt/tau); beta = 1 - rho */
          double d_dtt = 0.0;
          for (int m = 0; m < M; ++m) {
            dbeta[m] = dkap[m] * k.w[m];
            dw[m] = dkap[m] * k.beta[m];
            d_dtt += (k.rho[m] / in->tau[m]) * (dbeta[m] - drho[m]);
          }
          /* softmax backward for read (c) and write (w) weights */
          double sc = 0.0, sw = 0.0;
          for (int m = 0; m < M; ++m) { sc += k.c[m] * dc[m]; sw += k.w[m] * dw[m]; }
          double dal = 0.0;
          for (int m = 0; m < M; ++m) {
            dzc[m] = k.c[m] * (dc[m] - sc);
            dzw[m] = k.w[m] * (dw[m] - sw);
            dal -= (dzc[m] + dzw[m]) * log(in->tau[m]);
          }
          if (out->dread_logit) for (int m = 0; m < M; ++m) out->dread_logit[ith * M + m] = dzc[m];
          if (out->dwrite_logit) for (int m = 0; m < M; ++m) out->dwrite_logit[ith * M + m] = dzw[m];
          /* dtt = dt * s, s = lambda^(1/alpha) */
          const double lam = in->lambda ? in->lambda[ith] : 1.0;
          const double a = in->alpha[ith];
          const double ds = d_dtt * in->dt[ith];
          if (out->ddt) out->ddt[ith] = d_dtt * k.s;
          if (in->lambda) {
            if (out->dlambda) out->dlambda[ith] = ds * k.s / (a * lam);
            dal += ds * (-k.s * log(lam) / (a * a));
          } else if (out->dlambda) {
            out->dlambda[ith] = 0.0;
          }
          if (out->dalpha) out->dalpha[ith] = dal;
        }
      }
      if (out->dinit_state) memcpy(out->dinit_state + bh * MNP, Gs, sizeof(double) * MNP);
      dD_part[bh] = dD_acc;
#undef COEF
#undef TOK
    }
    free(ckpt);
    free(buf);
    free(Gs);
    free(scratch);
  }
  if (status) { free(dB_part); free(dC_part); free(dD_part); return status; }

  /* fixed-order reductions over the heads of each group */
  const int64_t hpg = H / G;
  if (out->dBm || out->dCm) {
#pragma omp parallel for
    for (int64_t bt = 0; bt < Bsz * L; ++bt) {
      const int64_t b = bt / L, t = bt % L;
      for (int64_t g = 0; g < G; ++g) {
        double *oB = out->dBm ? out->dBm + ((b * L + t) * G + g) * N : NULL;
        double *oC = out->dCm ? out->dCm + ((b * L + t) * G + g) * N : NULL;
        for (int64_t n = 0; n < N; ++n) {
          double sb = 0.0, sc = 0.0;
          for (int64_t j = 0; j < hpg; ++j) {
            const int64_t h = g * hpg + j, bh = b * H + h;
            sb += dB_part[(bh * L + t) * N + n];
            sc += dC_part[(bh * L + t) * N + n];
          }
          if (oB) oB[n] = sb;
          if (oC) oC[n] = sc;
        }
      }
    }
  }
  if (out->dD) {
    for (int64_t h = 0; h < H; ++h) {
      double s = 0.0;
      for (int64_t b = 0; b < Bsz; ++b) s += dD_part[b * H + h];
      out->dD[h] = s;
    }
  }
  free(dB_part);
  free(dC_part);
  free(dD_part);
  return 0;
}
