/*
 * agrl_oracle.c -- CPU reference ("oracle") for the fused policy-loss path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the benchmark's CPU
 * baseline do.  It shares no code, header or constant with the HIP path.
 *
 * Plain, slow, obviously correct:
 *   - advantage normalisation in IEEE fp32, one rounding per operation,
 *     in the fixed summation order written out in csum64() below;
 *   - log-softmax, clipped surrogate, loss and gradients in fp64 from the
 *     exact upcast of the bf16/fp32 inputs, by their plain definitions.
 * Threads only split independent outputs (tokens or vocabulary rows); every
 * sum runs in index order.  Build with -ffp-contract=off (no FMA fusion).
 *
 * Paper references (AgentRL, arXiv 2510.04206):
 *   token log-probability of an action    -- App. B.1, the factorisation of
 *                                            pi(a_t|s_t) over the action's tokens
 *   task/sample/group/trajectory indexing -- App. B.1 "Multi-Task Setting"
 *   GRPO group-relative advantage         -- App. B.2, GRPO objective; App. A
 *   task advantage normalisation          -- Sec. 3.2, the normalisation
 *                                            equation and the token-level set
 *   clipped surrogate, ratio              -- App. B.2 PPO objective; App. A
 *   token-level loss normalisation, eps_low/eps_high -- App. A, DAPO objective
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* fp32 helpers: each statement is one IEEE round-to-nearest operation.      */
/* volatile stops the compiler from keeping wider intermediates or fusing.   */
static float f_add(float a, float b) { volatile float r = a + b; return r; }
static float f_sub(float a, float b) { volatile float r = a - b; return r; }
static float f_mul(float a, float b) { volatile float r = a * b; return r; }
static float f_div(float a, float b) { volatile float r = a / b; return r; }
static float f_sqrt(float a) { volatile float r = sqrtf(a); return r; }

/*
 * csum64: the fixed fp32 summation order used for every advantage statistic.
 * The terms x[t] of the members of a segment (sel[t] != 0), t ascending, are
 * dealt to 64 accumulators by t mod 64; each accumulator adds its terms in
 * ascending t starting from +0.  The 64 partial sums are then combined by a
 * butterfly: for o = 32, 16, 8, 4, 2, 1 every accumulator l becomes
 * acc[l] + acc[l xor o].  The result is accumulator 0.  (Every accumulator
 * ends with the same bits because fp addition is commutative.)
 */
static float csum64(const float* x, const unsigned char* sel, int64_t n) {
  float acc[64];
  for (int l = 0; l < 64; ++l) acc[l] = 0.0f;
  for (int64_t t = 0; t < n; ++t)
    if (sel[t]) acc[t % 64] = f_add(acc[t % 64], x[t]);
  for (int o = 32; o >= 1; o >>= 1) {
    float nxt[64];
    for (int l = 0; l < 64; ++l) nxt[l] = f_add(acc[l], acc[l ^ o]);
    for (int l = 0; l < 64; ++l) acc[l] = nxt[l];
  }
  return acc[0];
}

/*
 * Advantage normalisation (returns 0, or -1 on an out-of-range id).
 *
 * 1. Counts.  n_tau = number of tokens t with traj_id[t] == tau and
 *    mask[t] == 1 (traj_id < 0 marks padding); N_i = sum of n_tau over the
 *    trajectories of task i.  Integer, exact.
 * 2. Group stage (when traj_group != NULL): GRPO's group-relative advantage,
 *    A_hat = (R - mean_g R) / (std_g R + eps), population std when ddof == 0
 *    (App. B.2 GRPO; App. A).  A group with size - ddof <= 0 gives 0.
 *    Without groups A_hat = R.
 * 3. Task stage (Sec. 3.2): mean and std of the set of token-level advantages
 *    of task i.  Every action token of trajectory tau carries A_hat_tau, so
 *    the set holds A_hat_tau with multiplicity n_tau:
 *      mu_i    = sum_tau n_tau A_hat_tau / N_i
 *      sigma_i = sqrt( sum_tau n_tau (A_hat_tau - mu_i)^2 / (N_i - ddof) )
 *      A_tilde = (A_hat - mu_i) / (sigma_i + eps)
 *    A task with N_i == 0 gets mu = sigma = 0 and A_tilde = 0; N_i - ddof <= 0
 *    gives sigma = 0.
 * 4. adv_tok[t] = A_tilde of traj_id[t] on action tokens, 0 elsewhere.
 */
static int task_adv_norm_impl(int64_t T_g, int32_t n_traj, int32_t n_task, int32_t n_group,
                              const int32_t* traj_id, const uint8_t* mask,
                              const int32_t* traj_task, const int32_t* traj_group,
                              const float* reward, int32_t ddof, float eps, int32_t drop_uniform,
                              int32_t* act_count, int64_t* task_count, float* task_mean,
                              float* task_std, float* adv_traj, float* adv_tok);

int oracle_task_adv_norm(int64_t T_g, int32_t n_traj, int32_t n_task, int32_t n_group,
                         const int32_t* traj_id, const uint8_t* mask,
                         const int32_t* traj_task, const int32_t* traj_group,
                         const float* reward, int32_t ddof, float eps,
                         int32_t* act_count, int64_t* task_count, float* task_mean,
                         float* task_std, float* adv_traj, float* adv_tok) {
  return task_adv_norm_impl(T_g, n_traj, n_task, n_group, traj_id, mask, traj_task, traj_group,
                            reward, ddof, eps, 0, act_count, task_count, task_mean, task_std,
                            adv_traj, adv_tok);
}

/*
 * With drop_uniform (DAPO's dynamic sampling, App. A: groups whose responses
 * are all correct or all incorrect carry no signal and are filtered out), a
 * GRPO group whose rewards are all equal (exact fp32 equality; a group of one
 * is such a group) is dropped: its trajectories get advantage 0 and their
 * tokens are left out of the task statistics (N_i, mu_i, sigma_i).
 * act_count still counts every trajectory's action tokens.
 */
int oracle_task_adv_norm_ext(int64_t T_g, int32_t n_traj, int32_t n_task, int32_t n_group,
                             const int32_t* traj_id, const uint8_t* mask,
                             const int32_t* traj_task, const int32_t* traj_group,
                             const float* reward, int32_t ddof, float eps, int32_t drop_uniform,
                             int32_t* act_count, int64_t* task_count, float* task_mean,
                             float* task_std, float* adv_traj, float* adv_tok) {
  if (drop_uniform && !traj_group) return -2;
  return task_adv_norm_impl(T_g, n_traj, n_task, n_group, traj_id, mask, traj_task, traj_group,
                            reward, ddof, eps, drop_uniform, act_count, task_count, task_mean,
                            task_std, adv_traj, adv_tok);
}

/*
 * Sequence-level aggregation (App. B.2, GRPO objective: the mean over the
 * responses of each response's token mean) as per-token weights of a packed
 * micro-batch: count[j] = action tokens of trajectory j in it, n_seq =
 * trajectories with count[j] > 0, w[t] = 1 / (n_seq * count[traj_id[t]]) on
 * every action token with traj_id >= 0 (the quotient in fp64, rounded once to
 * fp32), 0 on every other token.  Returns -1 (and skips the token) for a
 * traj_id >= n_traj.
 */
int oracle_sequence_mean_weights(int64_t T, int32_t n_traj, const int32_t* traj_id,
                                 const uint8_t* mask, int32_t* count, float* w) {
  int rc = 0;
  for (int32_t j = 0; j < n_traj; ++j) count[j] = 0;
  for (int64_t t = 0; t < T; ++t) {
    if (traj_id[t] >= n_traj) rc = -1;
    else if (traj_id[t] >= 0 && mask[t]) count[traj_id[t]] += 1;
  }
  int64_t n_seq = 0;
  for (int32_t j = 0; j < n_traj; ++j) n_seq += count[j] > 0;
  for (int64_t t = 0; t < T; ++t) {
    const int32_t j = traj_id[t];
    w[t] = (j >= 0 && j < n_traj && mask[t]) ? (float)(1.0 / ((double)n_seq * (double)count[j]))
                                             : 0.0f;
  }
  return rc;
}

static int task_adv_norm_impl(int64_t T_g, int32_t n_traj, int32_t n_task, int32_t n_group,
                              const int32_t* traj_id, const uint8_t* mask,
                              const int32_t* traj_task, const int32_t* traj_group,
                              const float* reward, int32_t ddof, float eps, int32_t drop_uniform,
                              int32_t* act_count, int64_t* task_count, float* task_mean,
                              float* task_std, float* adv_traj, float* adv_tok) {
  for (int32_t j = 0; j < n_traj; ++j) act_count[j] = 0;
  for (int64_t t = 0; t < T_g; ++t) {
    if (traj_id[t] >= n_traj) return -1;
    if (traj_id[t] >= 0 && mask[t]) act_count[traj_id[t]] += 1;
  }
  for (int32_t j = 0; j < n_traj; ++j) {
    if (traj_task[j] < 0 || traj_task[j] >= n_task) return -1;
    if (traj_group && (traj_group[j] < 0 || traj_group[j] >= n_group)) return -1;
  }

  float* a_hat = (float*)malloc(sizeof(float) * (size_t)(n_traj > 0 ? n_traj : 1));
  float* term = (float*)malloc(sizeof(float) * (size_t)(n_traj > 0 ? n_traj : 1));
  unsigned char* sel = (unsigned char*)malloc((size_t)(n_traj > 0 ? n_traj : 1));
  unsigned char* dropped = (unsigned char*)calloc((size_t)(n_traj > 0 ? n_traj : 1), 1);

  /* group stage */
  if (traj_group) {
    for (int32_t g = 0; g < n_group; ++g) {
      int32_t K = 0;
      for (int32_t j = 0; j < n_traj; ++j) {
        sel[j] = (traj_group[j] == g);
        K += sel[j];
      }
      if (K == 0) continue;
      if (drop_uniform) {
        int uniform = 1;
        float r0 = 0.0f;
        int seen = 0;
        for (int32_t j = 0; j < n_traj; ++j) {
          if (!sel[j]) continue;
          if (!seen) {
            r0 = reward[j];
            seen = 1;
          } else if (reward[j] != r0) {
            uniform = 0;
          }
        }
        if (uniform) {
          for (int32_t j = 0; j < n_traj; ++j)
            if (sel[j]) {
              dropped[j] = 1;
              a_hat[j] = 0.0f;
            }
          continue;
        }
      }
      if (K - ddof <= 0) {
        for (int32_t j = 0; j < n_traj; ++j)
          if (sel[j]) a_hat[j] = 0.0f;
        continue;
      }
      float mu = f_div(csum64(reward, sel, n_traj), (float)K);
      for (int32_t j = 0; j < n_traj; ++j) {
        float dv = f_sub(reward[j], mu);
        term[j] = f_mul(dv, dv);
      }
      float var = f_div(csum64(term, sel, n_traj), (float)(K - ddof));
      float den = f_add(f_sqrt(var), eps);
      for (int32_t j = 0; j < n_traj; ++j)
        if (sel[j]) a_hat[j] = f_div(f_sub(reward[j], mu), den);
    }
  } else {
    for (int32_t j = 0; j < n_traj; ++j) a_hat[j] = reward[j];
  }

  /* task stage */
  for (int32_t i = 0; i < n_task; ++i) {
    int64_t N = 0;
    for (int32_t j = 0; j < n_traj; ++j) {
      sel[j] = (traj_task[j] == i) && !dropped[j];
      if (sel[j]) N += act_count[j];
    }
    task_count[i] = N;
    if (N == 0) {
      task_mean[i] = 0.0f;
      task_std[i] = 0.0f;
      for (int32_t j = 0; j < n_traj; ++j)
        if (sel[j]) adv_traj[j] = 0.0f;
      continue;
    }
    for (int32_t j = 0; j < n_traj; ++j) term[j] = f_mul((float)act_count[j], a_hat[j]);
    float mu = f_div(csum64(term, sel, n_traj), (float)N);
    for (int32_t j = 0; j < n_traj; ++j) {
      float dv = f_sub(a_hat[j], mu);
      term[j] = f_mul((float)act_count[j], f_mul(dv, dv));
    }
    float sigma = 0.0f;
    if (N - ddof > 0) sigma = f_sqrt(f_div(csum64(term, sel, n_traj), (float)(N - ddof)));
    float den = f_add(sigma, eps);
    task_mean[i] = mu;
    task_std[i] = sigma;
    for (int32_t j = 0; j < n_traj; ++j)
      if (sel[j]) adv_traj[j] = f_div(f_sub(a_hat[j], mu), den);
  }
  for (int32_t j = 0; j < n_traj; ++j)
    if (dropped[j]) adv_traj[j] = 0.0f;

  if (adv_tok)
    for (int64_t t = 0; t < T_g; ++t)
      adv_tok[t] = (mask[t] && traj_id[t] >= 0) ? adv_traj[traj_id[t]] : 0.0f;

  free(a_hat);
  free(term);
  free(sel);
  free(dropped);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* fp64 policy loss                                                          */

/* element k of an input matrix stored as fp32 (is_bf16 == 0) or bf16 bits */
static double load_in(const void* p, int is_bf16, int64_t k) {
  if (is_bf16) {
    uint32_t u = (uint32_t)((const uint16_t*)p)[k] << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
  }
  return (double)((const float*)p)[k];
}

typedef struct {
  int64_t T;
  int32_t d, V, is_bf16;
  const void* H;
  const void* W;
  const int32_t* y;
  const uint8_t* mask;
  const float* adv;
  const float* old;
  double eps_lo, eps_hi, inv_temp, n_norm, grad_loss;
  /* per-token results of the forward (fp64) */
  double* lse;
  double* logp;
  double* g;          /* dL/dlogp */
  /* outputs */
  double* dH;
  double* dW;
  /* work split */
  const int64_t* rows; /* rows to process (tokens or vocabulary rows) */
  int64_t n_rows;
  int nthreads;
  int tid;
} job_t;

/* z_v = inv_temp * <h, w_v> for every v; h given upcast */
static void logits_row(const job_t* J, const double* h, double* z) {
  for (int32_t v = 0; v < J->V; ++v) {
    double acc = 0.0;
    for (int32_t k = 0; k < J->d; ++k) acc += h[k] * load_in(J->W, J->is_bf16, (int64_t)v * J->d + k);
    z[v] = acc * J->inv_temp;
  }
}

static void upcast_row(const job_t* J, int64_t n, double* h) {
  for (int32_t k = 0; k < J->d; ++k) h[k] = load_in(J->H, J->is_bf16, n * J->d + k);
}

/* lse_n = M + log sum_v exp(z_v - M), M = max_v z_v; logp_n = z_{y_n} - lse_n */
static void* fwd_worker(void* arg) {
  job_t* J = (job_t*)arg;
  double* h = (double*)malloc(sizeof(double) * (size_t)J->d);
  double* z = (double*)malloc(sizeof(double) * (size_t)J->V);
  for (int64_t r = J->tid; r < J->n_rows; r += J->nthreads) {
    int64_t n = J->rows[r];
    upcast_row(J, n, h);
    logits_row(J, h, z);
    double M = -INFINITY;
    for (int32_t v = 0; v < J->V; ++v) M = z[v] > M ? z[v] : M;
    double s = 0.0;
    for (int32_t v = 0; v < J->V; ++v) s += exp(z[v] - M);
    J->lse[n] = M + log(s);
    J->logp[n] = z[J->y[n]] - J->lse[n];
  }
  free(h);
  free(z);
  return NULL;
}

/* dH_n = inv_temp * g_n * (w_{y_n} - sum_v p_{n,v} w_v) */
static void* dh_worker(void* arg) {
  job_t* J = (job_t*)arg;
  double* h = (double*)malloc(sizeof(double) * (size_t)J->d);
  double* z = (double*)malloc(sizeof(double) * (size_t)J->V);
  double* acc = (double*)malloc(sizeof(double) * (size_t)J->d);
  for (int64_t r = J->tid; r < J->n_rows; r += J->nthreads) {
    int64_t n = J->rows[r];
    double* out = J->dH + r * J->d;
    if (!J->mask[n]) {
      for (int32_t k = 0; k < J->d; ++k) out[k] = 0.0;
      continue;
    }
    upcast_row(J, n, h);
    logits_row(J, h, z);
    for (int32_t k = 0; k < J->d; ++k) acc[k] = 0.0;
    for (int32_t v = 0; v < J->V; ++v) {
      double p = exp(z[v] - J->lse[n]);
      double c = (v == J->y[n] ? 1.0 : 0.0) - p;
      for (int32_t k = 0; k < J->d; ++k) acc[k] += c * load_in(J->W, J->is_bf16, (int64_t)v * J->d + k);
    }
    for (int32_t k = 0; k < J->d; ++k) out[k] = J->inv_temp * J->g[n] * acc[k];
  }
  free(h);
  free(z);
  free(acc);
  return NULL;
}

/* dW_v = inv_temp * sum_n g_n (1[v == y_n] - p_{n,v}) h_n, n over action tokens */
static void* dw_worker(void* arg) {
  job_t* J = (job_t*)arg;
  double* h = (double*)malloc(sizeof(double) * (size_t)J->d);
  double* w = (double*)malloc(sizeof(double) * (size_t)J->d);
  double* acc = (double*)malloc(sizeof(double) * (size_t)J->d);
  for (int64_t r = J->tid; r < J->n_rows; r += J->nthreads) {
    int64_t v = J->rows[r];
    for (int32_t k = 0; k < J->d; ++k) {
      w[k] = load_in(J->W, J->is_bf16, v * J->d + k);
      acc[k] = 0.0;
    }
    for (int64_t n = 0; n < J->T; ++n) {
      if (!J->mask[n]) continue;
      upcast_row(J, n, h);
      double zv = 0.0;
      for (int32_t k = 0; k < J->d; ++k) zv += h[k] * w[k];
      zv *= J->inv_temp;
      double p = exp(zv - J->lse[n]);
      double c = J->g[n] * ((v == J->y[n] ? 1.0 : 0.0) - p);
      for (int32_t k = 0; k < J->d; ++k) acc[k] += c * h[k];
    }
    double* out = J->dW + r * J->d;
    for (int32_t k = 0; k < J->d; ++k) out[k] = J->inv_temp * acc[k];
  }
  free(h);
  free(w);
  free(acc);
  return NULL;
}

static void run_threads(job_t* base, void* (*fn)(void*)) {
  int nt = base->nthreads < 1 ? 1 : base->nthreads;
  pthread_t* th = (pthread_t*)malloc(sizeof(pthread_t) * (size_t)nt);
  job_t* jobs = (job_t*)malloc(sizeof(job_t) * (size_t)nt);
  for (int i = 0; i < nt; ++i) {
    jobs[i] = *base;
    jobs[i].nthreads = nt;
    jobs[i].tid = i;
    pthread_create(&th[i], NULL, fn, &jobs[i]);
  }
  for (int i = 0; i < nt; ++i) pthread_join(th[i], NULL);
  free(th);
  free(jobs);
}

/*
 * Per-token surrogate and its derivative (App. B.2 PPO; App. A DAPO):
 *   rho = exp(logp - old)
 *   s   = min(rho A, clip(rho, 1 - eps_lo, 1 + eps_hi) A)
 *   L   = -(1 / N_norm) sum_n s_n            (minimised)
 *   g_n = dL/dlogp_n = -(grad_loss / N_norm) A rho   when the unclipped
 *         branch is the minimum, 0 when the clipped branch is strictly
 *         smaller (A > 0 and rho > 1 + eps_hi, or A < 0 and rho < 1 - eps_lo).
 * Returns s_n; writes g_n and the clip flag (+1 high, -1 low, 0 none).
 */
static double surrogate(double logp, double old, double A, double eps_lo, double eps_hi,
                        double scale, double* g, int* clip) {
  double rho = exp(logp - old);
  double rc = rho;
  if (rc < 1.0 - eps_lo) rc = 1.0 - eps_lo;
  if (rc > 1.0 + eps_hi) rc = 1.0 + eps_hi;
  double u = rho * A, c = rc * A;
  *clip = 0;
  if (A > 0.0 && rho > 1.0 + eps_hi) *clip = 1;
  if (A < 0.0 && rho < 1.0 - eps_lo) *clip = -1;
  *g = (*clip != 0) ? 0.0 : -scale * A * rho;
  return u < c ? u : c;
}

static void fill_job(job_t* J, int64_t T, int32_t d, int32_t V, int32_t is_bf16, const void* H,
                     const void* W, const int32_t* y, const uint8_t* mask, const float* adv,
                     const float* old, double eps_lo, double eps_hi, double inv_temp,
                     int nthreads) {
  memset(J, 0, sizeof *J);
  J->T = T;
  J->d = d;
  J->V = V;
  J->is_bf16 = is_bf16;
  J->H = H;
  J->W = W;
  J->y = y;
  J->mask = mask;
  J->adv = adv;
  J->old = old;
  J->eps_lo = eps_lo;
  J->eps_hi = eps_hi;
  J->inv_temp = inv_temp;
  J->nthreads = nthreads;
}

static int64_t* action_rows(int64_t T, const uint8_t* mask, int64_t* count) {
  int64_t c = 0;
  for (int64_t n = 0; n < T; ++n) c += mask[n] != 0;
  int64_t* r = (int64_t*)malloc(sizeof(int64_t) * (size_t)(c > 0 ? c : 1));
  c = 0;
  for (int64_t n = 0; n < T; ++n)
    if (mask[n]) r[c++] = n;
  *count = c;
  return r;
}

/*
 * KL penalty of a token against a reference policy (App. A: the PPO and GRPO
 * objectives subtract beta * D_KL).  With l = logp and r = ref_logp:
 *   estimator 0 (k3): KL = exp(r - l) - (r - l) - 1,  dKL/dl = 1 - exp(r - l)
 *   estimator 1 (k1): KL = l - r,                      dKL/dl = 1
 */
static double kl_term(double l, double r, int estimator, double* dkl) {
  if (estimator == 1) {
    *dkl = 1.0;
    return l - r;
  }
  double u = r - l;
  *dkl = 1.0 - exp(u);
  return exp(u) - u - 1.0;
}

/*
 * Forward (and, when dH/dW are given, backward) over the whole micro-batch.
 * n_norm <= 0 means N_norm = number of action tokens.  Masked tokens are
 * never read; their logp/lse outputs are 0 and their dH rows +0.
 * Outputs: logp[T], lse[T] (fp64), loss, n_clip[2] = {#clip high, #clip low},
 * g[T] = dL/dlogp (nullable), dH[T*d], dW[V*d] (nullable; fp64).
 *
 * Extensions (policy_loss_ext): per token f = s - kl_beta * KL(logp, ref_logp)
 * (KL as in kl_term; kl_beta == 0 leaves the surrogate alone), and per-token
 * weights w replacing 1 / N_norm when token_weight is given:
 *   L = -sum_n w_n f_n,   g_n = -grad_loss w_n (ds_n/dlogp - kl_beta dKL_n/dlogp).
 */
static int policy_loss_impl(int64_t T, int32_t d, int32_t V, int32_t is_bf16, const void* H,
                            const void* W, const int32_t* y, const uint8_t* mask,
                            const float* adv, const float* old, double eps_lo, double eps_hi,
                            int64_t n_norm, double temperature, double grad_loss,
                            double kl_beta, int kl_estimator, const float* ref_logp,
                            const float* token_weight, int nthreads, double* logp, double* lse,
                            double* loss, int64_t* n_clip, double* g, double* dH, double* dW);

int oracle_policy_loss(int64_t T, int32_t d, int32_t V, int32_t is_bf16, const void* H,
                       const void* W, const int32_t* y, const uint8_t* mask, const float* adv,
                       const float* old, double eps_lo, double eps_hi, int64_t n_norm,
                       double temperature, double grad_loss, int nthreads, double* logp,
                       double* lse, double* loss, int64_t* n_clip, double* g, double* dH,
                       double* dW) {
  return policy_loss_impl(T, d, V, is_bf16, H, W, y, mask, adv, old, eps_lo, eps_hi, n_norm,
                          temperature, grad_loss, 0.0, 0, NULL, NULL, nthreads, logp, lse, loss,
                          n_clip, g, dH, dW);
}

int oracle_policy_loss_ext(int64_t T, int32_t d, int32_t V, int32_t is_bf16, const void* H,
                           const void* W, const int32_t* y, const uint8_t* mask,
                           const float* adv, const float* old, double eps_lo, double eps_hi,
                           int64_t n_norm, double temperature, double grad_loss, double kl_beta,
                           int kl_estimator, const float* ref_logp, const float* token_weight,
                           int nthreads, double* logp, double* lse, double* loss,
                           int64_t* n_clip, double* g, double* dH, double* dW) {
  if (kl_beta != 0.0 && !ref_logp) return -2;
  return policy_loss_impl(T, d, V, is_bf16, H, W, y, mask, adv, old, eps_lo, eps_hi, n_norm,
                          temperature, grad_loss, kl_beta, kl_estimator, ref_logp, token_weight,
                          nthreads, logp, lse, loss, n_clip, g, dH, dW);
}

static int policy_loss_impl(int64_t T, int32_t d, int32_t V, int32_t is_bf16, const void* H,
                            const void* W, const int32_t* y, const uint8_t* mask,
                            const float* adv, const float* old, double eps_lo, double eps_hi,
                            int64_t n_norm, double temperature, double grad_loss,
                            double kl_beta, int kl_estimator, const float* ref_logp,
                            const float* token_weight, int nthreads, double* logp, double* lse,
                            double* loss, int64_t* n_clip, double* g, double* dH, double* dW) {
  for (int64_t n = 0; n < T; ++n)
    if (mask[n] && (y[n] < 0 || y[n] >= V)) return -1;
  job_t J;
  fill_job(&J, T, d, V, is_bf16, H, W, y, mask, adv, old, eps_lo, eps_hi, 1.0 / temperature,
           nthreads);
  int64_t n_act = 0;
  int64_t* rows = action_rows(T, mask, &n_act);
  double* gg = (double*)calloc((size_t)(T > 0 ? T : 1), sizeof(double));
  for (int64_t n = 0; n < T; ++n) logp[n] = lse[n] = 0.0;
  J.lse = lse;
  J.logp = logp;
  J.g = gg;
  J.rows = rows;
  J.n_rows = n_act;
  if (n_act > 0) run_threads(&J, fwd_worker);

  double N = (double)(n_norm > 0 ? n_norm : n_act);
  double sum = 0.0;
  int64_t hi = 0, lo = 0;
  for (int64_t r = 0; r < n_act; ++r) {
    int64_t n = rows[r];
    int clip;
    /* weight of the token: 1/N (applied after the sum) or the caller's w_n */
    double scale = token_weight ? grad_loss * (double)token_weight[n]
                                : (N > 0 ? grad_loss / N : 0.0);
    double f = surrogate(logp[n], (double)old[n], (double)adv[n], eps_lo, eps_hi, scale,
                         &gg[n], &clip);
    if (kl_beta != 0.0) {
      double dkl;
      f -= kl_beta * kl_term(logp[n], (double)ref_logp[n], kl_estimator, &dkl);
      gg[n] += scale * kl_beta * dkl;
    }
    sum += token_weight ? (double)token_weight[n] * f : f;
    hi += clip == 1;
    lo += clip == -1;
  }
  if (token_weight)
    *loss = -sum;
  else
    *loss = N > 0 ? -sum / N : 0.0;
  if (n_clip) {
    n_clip[0] = hi;
    n_clip[1] = lo;
  }
  if (g)
    for (int64_t n = 0; n < T; ++n) g[n] = gg[n];

  if (dH) {
    int64_t* all = (int64_t*)malloc(sizeof(int64_t) * (size_t)(T > 0 ? T : 1));
    for (int64_t n = 0; n < T; ++n) all[n] = n;
    J.rows = all;
    J.n_rows = T;
    J.dH = dH;
    run_threads(&J, dh_worker);
    free(all);
  }
  if (dW) {
    int64_t* vr = (int64_t*)malloc(sizeof(int64_t) * (size_t)(V > 0 ? V : 1));
    for (int32_t v = 0; v < V; ++v) vr[v] = v;
    J.rows = vr;
    J.n_rows = V;
    J.dW = dW;
    run_threads(&J, dw_worker);
    free(vr);
  }
  free(rows);
  free(gg);
  return 0;
}

/*
 * Sampled check at sizes where the whole batch is too slow for the CPU:
 * for the listed tokens only, lse/logp (fp64) and the dH row.  N_norm is the
 * action-token count of the whole micro-batch (or n_norm > 0), an integer
 * the oracle counts itself.  out_dH may be NULL.
 */
int oracle_token_sample(int64_t T, int32_t d, int32_t V, int32_t is_bf16, const void* H,
                        const void* W, const int32_t* y, const uint8_t* mask, const float* adv,
                        const float* old, double eps_lo, double eps_hi, int64_t n_norm,
                        double temperature, double grad_loss, int nthreads,
                        const int64_t* tokens, int64_t n_tokens, double* out_lse,
                        double* out_logp, double* out_g, double* out_dH) {
  for (int64_t i = 0; i < n_tokens; ++i) {
    int64_t n = tokens[i];
    if (n < 0 || n >= T) return -1;
    if (mask[n] && (y[n] < 0 || y[n] >= V)) return -1;
  }
  int64_t n_act = 0;
  for (int64_t n = 0; n < T; ++n) n_act += mask[n] != 0;
  double N = (double)(n_norm > 0 ? n_norm : n_act);
  job_t J;
  fill_job(&J, T, d, V, is_bf16, H, W, y, mask, adv, old, eps_lo, eps_hi, 1.0 / temperature,
           nthreads);
  /* the forward writes lse/logp at token index n: use T-sized scratch */
  double* lse = (double*)calloc((size_t)(T > 0 ? T : 1), sizeof(double));
  double* logp = (double*)calloc((size_t)(T > 0 ? T : 1), sizeof(double));
  double* gg = (double*)calloc((size_t)(T > 0 ? T : 1), sizeof(double));
  int64_t* act = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n_tokens > 0 ? n_tokens : 1));
  int64_t na = 0;
  for (int64_t i = 0; i < n_tokens; ++i)
    if (mask[tokens[i]]) act[na++] = tokens[i];
  J.lse = lse;
  J.logp = logp;
  J.g = gg;
  J.rows = act;
  J.n_rows = na;
  if (na > 0) run_threads(&J, fwd_worker);
  for (int64_t i = 0; i < na; ++i) {
    int64_t n = act[i];
    int clip;
    surrogate(logp[n], (double)old[n], (double)adv[n], eps_lo, eps_hi,
              N > 0 ? grad_loss / N : 0.0, &gg[n], &clip);
  }
  for (int64_t i = 0; i < n_tokens; ++i) {
    int64_t n = tokens[i];
    out_lse[i] = lse[n];
    out_logp[i] = logp[n];
    if (out_g) out_g[i] = gg[n];
  }
  if (out_dH) {
    J.rows = tokens;
    J.n_rows = n_tokens;
    J.dH = out_dH;
    run_threads(&J, dh_worker);
  }
  free(lse);
  free(logp);
  free(gg);
  free(act);
  return 0;
}

/*
 * The surrogate, loss and dL/dlogp of every action token from log-probs the
 * caller already holds (App. B.2 PPO objective; App. A DAPO token-level
 * normalisation): the second half of the whole-batch forward above, for
 * batches whose log-probs come from the fp64 full-logit pass in blas.py.
 * logp is fp64 [T] (read on action tokens).  Outputs loss, n_clip[2] and
 * g[T] (0 on masked tokens).
 */
int oracle_surrogate_terms(int64_t T, const uint8_t* mask, const float* adv, const float* old,
                           const double* logp, double eps_lo, double eps_hi, int64_t n_norm,
                           double grad_loss, double* loss, int64_t* n_clip, double* g) {
  int64_t n_act = 0;
  for (int64_t n = 0; n < T; ++n) n_act += mask[n] != 0;
  double N = (double)(n_norm > 0 ? n_norm : n_act);
  double sum = 0.0;
  int64_t hi = 0, lo = 0;
  for (int64_t n = 0; n < T; ++n) {
    g[n] = 0.0;
    if (!mask[n]) continue;
    int clip;
    sum += surrogate(logp[n], (double)old[n], (double)adv[n], eps_lo, eps_hi,
                     N > 0 ? grad_loss / N : 0.0, &g[n], &clip);
    hi += clip == 1;
    lo += clip == -1;
  }
  *loss = N > 0 ? -sum / N : 0.0;
  n_clip[0] = hi;
  n_clip[1] = lo;
  return 0;
}

/*
 * Rows of dW for the listed vocabulary entries, given every action token's
 * lse and dL/dlogp (as produced above): dW_v = sum_n g_n (1[v == y_n] - p_{n,v}) h_n
 * over action tokens n, by the same per-row pass as the whole-batch backward.
 * out_dW is [n_rows, d] fp64.
 */
int oracle_dw_rows(int64_t T, int32_t d, int32_t V, int32_t is_bf16, const void* H,
                   const void* W, const int32_t* y, const uint8_t* mask, double temperature,
                   const double* lse, const double* g, const int64_t* rows, int64_t n_rows,
                   int nthreads, double* out_dW) {
  for (int64_t i = 0; i < n_rows; ++i)
    if (rows[i] < 0 || rows[i] >= V) return -1;
  for (int64_t n = 0; n < T; ++n)
    if (mask[n] && (y[n] < 0 || y[n] >= V)) return -1;
  job_t J;
  fill_job(&J, T, d, V, is_bf16, H, W, y, mask, NULL, NULL, 0.0, 0.0, 1.0 / temperature,
           nthreads);
  J.lse = (double*)lse;
  J.g = (double*)g;
  J.rows = rows;
  J.n_rows = n_rows;
  J.dW = out_dW;
  run_threads(&J, dw_worker);
  return 0;
}
